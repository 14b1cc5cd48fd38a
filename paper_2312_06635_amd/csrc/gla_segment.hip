// gla_segment.hip -- sequence parallelism for few heads and long sequences
// (the two-stage scan of App. A.2 over segments of whole chunks).  A head's
// sequence [T] is viewed as nseg segments of T/nseg steps, which the kernels
// treat as independent heads; these kernels connect them.  With D_s the decay
// of segment s (the product of its chunk decays gamma, per key feature):
//   forward:  S_in[0] = S0,  S_in[s+1] = Diag(D_s) S_in[s] + S_loc[s]
//             (S_loc[s]: segment s's final state from a zero initial state;
//             S_in[nseg] is the head's S_T);
//   backward: dS_out[nseg-1] = dS_T,  dS_out[s-1] = Diag(D_s) dS_out[s] + dS0_loc[s]
//             (dS0_loc[s]: the gradient of segment s's initial state from a
//             zero final-state gradient; the head's dS0 continues one more step).
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

// dec[seg][k] = product of the segment's chunk decays.
__global__ void __launch_bounds__(256) seg_decay_kernel(const float *gam, float *dec, int64_t n, int Ns, int K) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t seg = i / K;
  const int k = (int)(i - seg * K);
  const float *g = gam + seg * Ns * K + k;
  float d = 1.f;
  for (int c = 0; c < Ns; ++c) d *= g[(int64_t)c * K];
  dec[i] = d;
}

// Thread per (head, key feature, value column) element of the state.
__global__ void __launch_bounds__(256) seg_fwd_scan_kernel(const float *dec, const float *S0, const float *Sloc,
                                                           float *Sin, float *ST, int64_t n, int nseg, int K,
                                                           int V) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t KV = (int64_t)K * V, bh = i / KV, e = i - bh * KV;
  const int k = (int)(e / V);
  float S = S0 ? S0[i] : 0.f;
  for (int s = 0; s < nseg; ++s) {
    const int64_t seg = bh * nseg + s;
    Sin[seg * KV + e] = S;
    S = dec[seg * K + k] * S + Sloc[seg * KV + e];
  }
  if (ST) ST[i] = S;
}

__global__ void __launch_bounds__(256) seg_bwd_scan_kernel(const float *dec, const float *dST, const float *dS0loc,
                                                           float *dSout, float *dS0, int64_t n, int nseg, int K,
                                                           int V) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int64_t KV = (int64_t)K * V, bh = i / KV, e = i - bh * KV;
  const int k = (int)(e / V);
  float D = dST ? dST[i] : 0.f;
  for (int s = nseg - 1; s >= 0; --s) {
    const int64_t seg = bh * nseg + s;
    dSout[seg * KV + e] = D;
    D = dec[seg * K + k] * D + dS0loc[seg * KV + e];
  }
  if (dS0) dS0[i] = D;
}

unsigned blocks_of(int64_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace

hipError_t launch_seg_decay(const Shape &s2, const float *gam, float *dec, hipStream_t st) {
  const int64_t n = (int64_t)s2.BH * s2.K;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(seg_decay_kernel, dim3(blocks_of(n)), dim3(256), 0, st, gam, dec, n, s2.N, s2.K);
  return hipGetLastError();
}

hipError_t launch_seg_fwd_scan(int BH, int nseg, int K, int V, const float *dec, const float *S0, const float *Sloc,
                               float *Sin, float *ST, hipStream_t st) {
  const int64_t n = (int64_t)BH * K * V;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(seg_fwd_scan_kernel, dim3(blocks_of(n)), dim3(256), 0, st, dec, S0, Sloc, Sin, ST, n, nseg, K,
                     V);
  return hipGetLastError();
}

hipError_t launch_seg_bwd_scan(int BH, int nseg, int K, int V, const float *dec, const float *dST,
                               const float *dS0loc, float *dSout, float *dS0, hipStream_t st) {
  const int64_t n = (int64_t)BH * K * V;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(seg_bwd_scan_kernel, dim3(blocks_of(n)), dim3(256), 0, st, dec, dST, dS0loc, dSout, dS0, n,
                     nseg, K, V);
  return hipGetLastError();
}

}  // namespace gla
