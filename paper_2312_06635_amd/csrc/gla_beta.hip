// gla_beta.hip -- value-side gate of the general form (App. C, G_t =
// alpha_t^T beta_t) in the backward: the chunk-local operands the sweeps use
// and the gate gradient
//     dlog beta_t = sum_{i >= t} (o_i (.) do_i - v_i (.) dv_i) + colsum(S_T (.) dS_T).
// The part of that sum beyond chunk n equals colsum(S_[n+1] (.) dS_[n+1])
// exactly (the state-form gate gradient at the next chunk's first step), so
// the carry into each chunk comes from the chunk-end states (summed over the
// key tiles by the dk sweep) and only the chunk's own rows are summed here:
// no rounding accumulates over the sequence.
// With E the chunk-local inclusive cumsum of log beta per value column,
//     Vh = V (.) exp(-E),   Oh = dO (.) exp(E),   gb = exp(E_last) per chunk,
// the backward sweeps keep the structure of the alpha-only layer (dP = Oh Vh^T
// masked, dq from Oh S^T, dk from Vh (dS gb)^T, the state columns decaying by
// gb).  Every kernel here is elementwise along value columns: a thread owns
// one (batch-head, chunk, value column) and walks the chunk's rows, so loads
// and stores are coalesced across threads.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

struct BetaArgs {
  const void *v, *dO, *lb, *o, *dv;
  void *Vh, *Oh, *dlb;
  float *gb;
  const float *cpart;     // [BH][N][KT][V] per key tile colsum(S_[n+1] (.) dS_[n+1])
  int64_t n;              // BH N V threads
  int T, V, C, N, KT;
};

struct Cell {
  int64_t base;  // element offset of the chunk's first row in this column
  int64_t cn;    // (bh, chunk) index
  int rows, col;
};

__device__ __forceinline__ Cell cell_of(const BetaArgs &a, int64_t i) {
  Cell c;
  c.col = (int)(i % a.V);
  const int64_t r = i / a.V;
  const int n = (int)(r % a.N);
  const int64_t bh = r / a.N;
  const int t0 = n * a.C;
  c.rows = min(a.C, a.T - t0);
  c.base = (bh * a.T + t0) * a.V + c.col;
  c.cn = bh * a.N + n;
  return c;
}

template <typename T>
__global__ void __launch_bounds__(256) beta_prep_kernel(BetaArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.n) return;
  const Cell c = cell_of(a, i);
  const T *lb = (const T *)a.lb + c.base, *v = (const T *)a.v + c.base, *dO = (const T *)a.dO + c.base;
  T *Vh = (T *)a.Vh + c.base, *Oh = (T *)a.Oh + c.base;
  constexpr int RB = 8;  // rows whose loads are issued together
  float E = 0.f;
  for (int r0 = 0; r0 < c.rows; r0 += RB) {
    float x[RB], y[RB], z[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const bool ok = r0 + r < c.rows;
      const int64_t o = (int64_t)(ok ? r0 + r : r0) * a.V;
      x[r] = ok ? (float)lb[o] : 0.f;
      y[r] = (float)v[o];
      z[r] = (float)dO[o];
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      E += x[r];
      if (r0 + r < c.rows) {
        const int64_t o = (int64_t)(r0 + r) * a.V;
        Vh[o] = cvt<T>(y[r] * __expf(-E));
        Oh[o] = cvt<T>(z[r] * __expf(E));
      }
    }
  }
  a.gb[c.cn * a.V + c.col] = __expf(E);
}

// Reverse cumsum inside each chunk, starting from the chunk's carry (key
// tiles added in order).
template <typename T>
__global__ void __launch_bounds__(256) beta_grad_scan_kernel(BetaArgs a) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= a.n) return;
  const Cell c = cell_of(a, i);
  float carry = 0.f;
  for (int kt = 0; kt < a.KT; ++kt) carry += a.cpart[(c.cn * a.KT + kt) * a.V + c.col];
  const T *o = (const T *)a.o + c.base, *dO = (const T *)a.dO + c.base;
  const T *v = (const T *)a.v + c.base, *dv = (const T *)a.dv + c.base;
  T *dlb = (T *)a.dlb + c.base;
  for (int r = c.rows - 1; r >= 0; --r) {
    const int64_t e = (int64_t)r * a.V;
    carry += (float)o[e] * (float)dO[e] - (float)v[e] * (float)dv[e];
    dlb[e] = cvt<T>(carry);
  }
}

template <typename T>
hipError_t beta_launch(int which, const BetaArgs &a, hipStream_t st) {
  const unsigned blocks = (unsigned)((a.n + 255) / 256);
  if (which == 0) hipLaunchKernelGGL(beta_prep_kernel<T>, dim3(blocks), dim3(256), 0, st, a);
  if (which == 2) hipLaunchKernelGGL(beta_grad_scan_kernel<T>, dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

BetaArgs beta_args(const Shape &s) {
  BetaArgs a{};
  a.n = (int64_t)s.BH * s.N * s.V;
  a.T = s.T; a.V = s.V; a.C = s.C; a.N = s.N; a.KT = (s.K + 31) / 32;
  return a;
}

}  // namespace

hipError_t launch_beta_prep(const Shape &s, const void *v, const void *dO, const void *lb, const Work &w,
                            hipStream_t st) {
  BetaArgs a = beta_args(s);
  a.v = v; a.dO = dO; a.lb = lb; a.Vh = w.Vh; a.Oh = w.Oh; a.gb = w.gb;
  if (a.n == 0) return hipSuccess;
  return s.io == IO_BF16 ? beta_launch<bf16>(0, a, st) : beta_launch<float>(0, a, st);
}

hipError_t launch_beta_grad(const Shape &s, const void *o, const void *dO, const void *v, const void *dv,
                            void *dlb, const Work &w, hipStream_t st) {
  BetaArgs a = beta_args(s);
  a.o = o; a.dO = dO; a.v = v; a.dv = dv; a.dlb = dlb; a.cpart = w.cpart;
  if (a.n == 0) return hipSuccess;
  return s.io == IO_BF16 ? beta_launch<bf16>(2, a, st) : beta_launch<float>(2, a, st);
}

}  // namespace gla
