// gla_fwd.hip -- forward state pass + chunk output of the chunkwise GLA form,
// and the step-by-step recurrent forward.
//
// fwd_main: one workgroup per (head, tile of Tv value columns), sequential
// over the chunks (the non-materialised state pass of Sec. 3.3 / App. B,
// Alg. 5).  Wave w keeps the fp32 state columns S[:, 16w .. 16w+16) of the
// tile in matrix-core accumulators for the whole sequence.  The columns of S
// evolve independently (the gate of Eq. 3 scales rows), so no state is shared
// between workgroups.  For each chunk n, with the operands made by prep:
//   O_n     = (Q (.) Lambda)_n S_[n] + P_n V_n          (Sec. 4.2; P holds the
//                                                        intra-chunk part)
//   S_[n+1] = Diag(gamma_n) S_[n] + (K (.) Gamma)_n^T V_n
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

static int round_up(int x, int m) { return (x + m - 1) / m * m; }
// Smallest power of two >= max(x, lo) (tile widths must be powers of two).
static int pow2_at_least(int x, int lo) {
  int p = lo;
  while (p < x) p *= 2;
  return p;
}

struct MainArgs {
  const void *Qt, *Kt, *P, *v;
  const float *gam, *S0;
  void *o;
  float *ST;
  int BH, T, K, Kp, V, C, Cp, N, Tv, ntiles, ldk, ldv, ldp;
};

template <typename T, int KBP>
__global__ void __launch_bounds__(256) fwd_main_kernel(MainArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int NQ = sizeof(T) == 2 ? (KBP / 2 > 0 ? KBP / 2 : 1) : KBP;  // Q/K tile vectors per thread
  constexpr int NX = sizeof(T) == 2 ? 2 : 4;                             // V and P tiles
  int bh, tile;
  xcd_map(a.BH, a.ntiles, bh, tile);
  const int w = wave_id(), l = lane_id(), g = l >> 4, j = l & 15;
  const int K = a.K, V = a.V, C = a.C, Cp = a.Cp, Kp = a.Kp;
  const int ldk = a.ldk, ldv = a.ldv, ldp = a.ldp;
  const int v0 = tile * a.Tv;
  const bool active = 16 * w < a.Tv;  // waves beyond the tile width only help with loads
  const int col = v0 + 16 * w + j;
  const bool colv = active && col < V;
  T *sQ = (T *)smem;
  T *sK = sQ + Cp * ldk;
  T *sV = sK + Cp * ldk;
  T *sP = sV + Cp * ldv;
  float *sGam = (float *)(sP + C * ldp);

  f4 S[KBP];
#pragma unroll
  for (int kb = 0; kb < KBP; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kr = 16 * kb + 4 * g + r;
      S[kb][r] = (a.S0 && kr < K && colv) ? a.S0[((int64_t)bh * K + kr) * V + col] : 0.f;
    }

  const T *Qt = (const T *)a.Qt, *Kt = (const T *)a.Kt, *Pm = (const T *)a.P;
  const T *vin = (const T *)a.v;
  T *o = (T *)a.o;
  TileRegs<T, NQ> pq, pk;
  TileRegs<T, NX> pv, pp;
  float pg = 0.f;
  const T *Qh = Qt + (int64_t)bh * a.T * K, *Kh = Kt + (int64_t)bh * a.T * K;
  const T *vh = vin + (int64_t)bh * a.T * V + v0, *Ph = Pm + (int64_t)bh * a.N * C * C;
  const float *gh = a.gam + (int64_t)bh * a.N * K;
  auto load_chunk = [&](int n) {
    const int rv = min(C, a.T - n * C);
    pq.load(Qh + n * C * K, K, Cp, Kp, rv, K);
    pk.load(Kh + n * C * K, K, Cp, Kp, rv, K);
    pv.load(vh + n * C * V, V, Cp, a.Tv, rv, V - v0);
    pp.load(Ph + n * C * C, C, C, Cp, C, C);
    pg = (int)threadIdx.x < K ? gh[n * K + threadIdx.x] : 0.f;
  };
  load_chunk(0);
  for (int n = 0; n < a.N; ++n) {
    const int t0 = n * C, rv = min(C, a.T - t0);
    const int64_t rb = (int64_t)bh * a.T + t0;
    pq.store(sQ, ldk, Cp, Kp);
    pk.store(sK, ldk, Cp, Kp);
    pv.store(sV, ldv, Cp, a.Tv);
    pp.store(sP, ldp, C, Cp);
    if ((int)threadIdx.x < Kp) sGam[threadIdx.x] = pg;
    __syncthreads();
    if (n + 1 < a.N) load_chunk(n + 1);

    if (active) {
      const int nI = C / 16;
      f4 acc[4] = {zero4(), zero4(), zero4(), zero4()};
#pragma unroll
      for (int s = 0; s < KBP / 2; ++s) {
        const frag_t<T> bs = acc_frag<T>(S[2 * s], S[2 * s + 1]);
#pragma unroll
        for (int I = 0; I < 4; ++I)
          if (I < nI) acc[I] = mma<T>(acc[I], ld_row_perm<T>(sQ, ldk, 16 * I, 32 * s), bs);
      }
#pragma unroll
      for (int I = 0; I < 4; ++I) {
        if (I >= nI) continue;
        const int js = (16 * I + 16 + 31) >> 5;
        for (int s = 0; s < js; ++s)
          acc[I] = mma<T>(acc[I], ld_row<T>(sP, ldp, 16 * I, 32 * s), ld_col<T>(sV, ldv, 32 * s, 16 * w));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 16 * I + 4 * g + r;
          if (row < rv && colv) o[(rb + row) * V + col] = cvt<T>(acc[I][r]);
        }
      }
#pragma unroll
      for (int kb = 0; kb < KBP; ++kb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) S[kb][r] *= sGam[16 * kb + 4 * g + r];
        for (int s = 0; s < Cp / 32; ++s)
          S[kb] = mma<T>(S[kb], ld_col<T>(sK, ldk, 32 * s, 16 * kb), ld_col<T>(sV, ldv, 32 * s, 16 * w));
      }
    }
    __syncthreads();
  }
  if (a.ST && colv) {
#pragma unroll
    for (int kb = 0; kb < KBP; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kr = 16 * kb + 4 * g + r;
        if (kr < K) a.ST[((int64_t)bh * K + kr) * V + col] = S[kb][r];
      }
  }
}

static void main_geometry(const Shape &s, int &Kp, int &Cp, int &Tv, int &ldk, int &ldv, int &ldp) {
  Kp = pow2_at_least(s.K, 32);
  Cp = round_up(s.C, 32);
  Tv = pow2_at_least(s.V < 64 ? s.V : 64, 16);
  const int pad = 32 / s.esz();
  ldk = Kp + pad;
  ldv = Tv + pad;
  ldp = Cp + pad;
}

size_t lds_fwd_main(const Shape &s) {
  int Kp, Cp, Tv, ldk, ldv, ldp;
  main_geometry(s, Kp, Cp, Tv, ldk, ldv, ldp);
  return (size_t)s.esz() * (2 * Cp * ldk + Cp * ldv + Cp * ldp) + (size_t)Kp * sizeof(float);
}

template <typename T, int KBP>
static hipError_t launch_main_t(const MainArgs &a, int waves, size_t lds, hipStream_t st) {
  static bool attr = false;
  if (!attr) {
    hipFuncSetAttribute((const void *)fwd_main_kernel<T, KBP>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr = true;
  }
  hipLaunchKernelGGL((fwd_main_kernel<T, KBP>), dim3(a.BH * a.ntiles), dim3(64 * waves), lds, st, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t dispatch_main(const MainArgs &a, int waves, size_t lds, hipStream_t st) {
  switch (a.Kp / 16) {
    case 2: return launch_main_t<T, 2>(a, waves, lds, st);
    case 4: return launch_main_t<T, 4>(a, waves, lds, st);
    case 8: return launch_main_t<T, 8>(a, waves, lds, st);
    default: return launch_main_t<T, 16>(a, waves, lds, st);
  }
}

hipError_t launch_fwd_main(const Shape &s, const void *v, const float *S0, void *o, float *ST,
                           const Work &w, hipStream_t st) {
  MainArgs a;
  a.Qt = w.Qt; a.Kt = w.Kt; a.P = w.P; a.v = v; a.gam = w.gam; a.S0 = S0; a.o = o; a.ST = ST;
  a.BH = s.BH; a.T = s.T; a.K = s.K; a.V = s.V; a.C = s.C; a.N = s.N;
  main_geometry(s, a.Kp, a.Cp, a.Tv, a.ldk, a.ldv, a.ldp);
  a.ntiles = (s.V + a.Tv - 1) / a.Tv;
  const size_t lds = lds_fwd_main(s);
  return s.io == IO_BF16 ? dispatch_main<bf16>(a, 4, lds, st) : dispatch_main<float>(a, 4, lds, st);
}

// ------------------------------------------------------------- recurrent form
// Eq. 3 one step at a time.  Workgroup = (64 value columns, head); thread
// (column, quarter) holds the fp32 state rows of its quarter of d_k for its
// column; o_t is the sum of the four quarters' partial dot products.
struct RecArgs {
  const void *q, *k, *v, *la;
  const float *S0;
  void *o;
  float *ST;
  int T, K, V;
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
  const T *la = (const T *)a.la + (int64_t)bh * a.T * K, *v = (const T *)a.v + (int64_t)bh * a.T * V;
  T *o = (T *)a.o + (int64_t)bh * a.T * V;
  for (int t = 0; t < a.T; ++t) {
    for (int i = tid; i < K; i += 256) {
      sq[i] = (float)q[(int64_t)t * K + i];
      sk[i] = (float)k[(int64_t)t * K + i];
      sa[i] = __expf((float)la[(int64_t)t * K + i]);
    }
    const float vt = colv ? (float)v[(int64_t)t * V + col] : 0.f;
    __syncthreads();
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      const int kr = qt * KQ + i;
      if (i < KQ && kr < K) {
        S[i] = sa[kr] * S[i] + sk[kr] * vt;
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
                            const void *la, const float *S0, void *o, float *ST, hipStream_t st) {
  RecArgs a{q, k, v, la, S0, o, ST, s.T, s.K, s.V};
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
