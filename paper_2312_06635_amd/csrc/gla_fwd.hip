// gla_fwd.hip -- the step-by-step recurrent forward (Sec. 4.1, Eq. 3; with
// the value-side gate of App. C, G_t = alpha_t^T beta_t) and the T = 0 state
// copy.  The chunkwise state pass lives in gla_vsweep.hip.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

// ------------------------------------------------------------- recurrent form
// Eq. 3 one step at a time.  Workgroup = (64 value columns, head); thread
// (column, quarter) holds the fp32 state rows of its quarter of d_k for its
// column; o_t is the sum of the four quarters' partial dot products.
struct RecArgs {
  const void *q, *k, *v, *la, *lb;  // lb: log beta [BH][T][V], value-side gate (nullable)
  const float *S0;
  void *o;
  float *ST;
  int T, K, V;
  int sg;         // scalar gate: la is [BH][T], one value per step shared by every feature
  float inv_tau;  // gate epilogue (0: la holds log alpha)
};

template <typename T>
__global__ void __launch_bounds__(256) recurrent_kernel(RecArgs a) {
  __shared__ float sq[256], sk[256], sa[256], so[4][64];
  const int bh = blockIdx.y, tid = threadIdx.x, c = tid & 63, qt = tid >> 6;
  const int K = a.K, V = a.V, KQ = (K + 3) / 4;
  const int col = blockIdx.x * 64 + c;
  const bool colv = col < V;
  float S[64];
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    const int kr = qt * KQ + i;
    S[i] = (a.S0 && i < KQ && kr < K && colv) ? a.S0[((int64_t)bh * K + kr) * V + col] : 0.f;
  }
  const T *q = (const T *)a.q + (int64_t)bh * a.T * K, *k = (const T *)a.k + (int64_t)bh * a.T * K;
  const int lrow = a.sg ? 1 : K, lf = a.sg ? 0 : 1;  // gate elements per step, per feature
  const T *la = (const T *)a.la + (int64_t)bh * a.T * lrow, *v = (const T *)a.v + (int64_t)bh * a.T * V;
  const T *lb = (const T *)a.lb + (int64_t)bh * a.T * V;
  T *o = (T *)a.o + (int64_t)bh * a.T * V;
  for (int t = 0; t < a.T; ++t) {
    for (int i = tid; i < K; i += 256) {
      sq[i] = (float)q[(int64_t)t * K + i];
      sk[i] = (float)k[(int64_t)t * K + i];
      sa[i] = a.la ? __expf(gate_la((float)la[(int64_t)t * lrow + i * lf], a.inv_tau, true)) : 1.f;  // no gate: alpha = 1
    }
    const float vt = colv ? (float)v[(int64_t)t * V + col] : 0.f;
    // general gate (App. C): the value-side factor of this thread's column
    const float bt = (a.lb && colv) ? __expf((float)lb[(int64_t)t * V + col]) : 1.f;
    __syncthreads();
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      const int kr = qt * KQ + i;
      if (i < KQ && kr < K) {
        S[i] = sa[kr] * bt * S[i] + sk[kr] * vt;
        part += sq[kr] * S[i];
      }
    }
    so[qt][c] = part;
    __syncthreads();
    if (qt == 0 && colv) o[(int64_t)t * V + col] = cvt<T>(so[0][c] + so[1][c] + so[2][c] + so[3][c]);
  }
  if (a.ST) {
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      const int kr = qt * KQ + i;
      if (i < KQ && kr < K && colv) a.ST[((int64_t)bh * K + kr) * V + col] = S[i];
    }
  }
}

hipError_t launch_recurrent(const Shape &s, const void *q, const void *k, const void *v,
                            const void *la, const void *lb, const float *S0, void *o, float *ST, hipStream_t st) {
  RecArgs a{q, k, v, la, lb, S0, o, ST, s.T, s.K, s.V, s.sgate ? 1 : 0, s.inv_tau};
  dim3 grid((s.V + 63) / 64, s.BH);
  if (s.io == IO_BF16)
    hipLaunchKernelGGL(recurrent_kernel<bf16>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(recurrent_kernel<float>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

__global__ void copy_state_kernel(int64_t n, const float *src, float *dst) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src ? src[i] : 0.f;
}

hipError_t launch_copy_state(int64_t n, const float *src, float *dst, hipStream_t st) {
  if (n <= 0 || !dst) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  hipLaunchKernelGGL(copy_state_kernel, dim3(blocks), dim3(256), 0, st, n, src, dst);
  return hipGetLastError();
}

}  // namespace gla
