// gla_prep.hip -- per-chunk gate factors, gated operands and the intra-chunk
// matrix P of the chunkwise GLA form (paper Sec. 4.2 and 4.3).
//
// One workgroup per (chunk, head); wave w owns the 16-row block w of the
// chunk and each lane owns the features k = FPL lane .. +FPL-1.  With B the
// chunk-local inclusive cumsum of log alpha (so exp(B) = b_t / b_{chunk start}):
//   Qt    = q (.) exp(B)              (Q (.) Lambda)
//   Kt    = k (.) exp(B_last - B)      (K (.) Gamma)
//   gamma = exp(B_last)                (chunk decay)
//   P[i][j] = sum_k q_ik k_jk exp(B_ik - B_jk) for j <= i, else 0  (Eq. 4)
// P is tiled in 16x16 blocks (I, J):
//   * I > J ("orange", between sub-chunks): a bf16 (fp32 for fp32 io)
//     matrix-core product of operands normalised at block boundaries, so that
//     every exponent is <= 0:
//       (q_I (.) exp(B - z_I)) diag(exp(z_I - zend_J)) (k_J (.) exp(zend_J - B))^T
//     with z_I the log decay at the start of block I and zend_J at the end of J.
//   * I = J ("pink", inside a sub-chunk): Eq. 4 itself in fp32 on the vector
//     ALUs, one exponential of the log-space difference B_ik - B_jk per pair
//     and feature (Sec. 4.3: full precision, no division by a cumulative
//     decay), the partial sums of a lane's features then reduced across the
//     wave.  Any gate, however steep, is exact here: every exponent is <= 0.
// Sub-chunks shorter than 16 (c < 16) lie inside the diagonal blocks, whose
// fp32 evaluation is the same for any such c.
#include <type_traits>

#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

struct PrepArgs {
  const void *q, *k, *la;
  void *Qt, *Kt, *P;
  float *gam;
  int T, K, Kp, C, N, ldk;
  int sg;         // scalar gate: la is [BH][T], one value per step shared by every feature
  float inv_tau;  // gate epilogue (0: la holds log alpha)
};

// Entry e of a 16x16 lower triangle (diagonal included), row-major.
__host__ __device__ constexpr int tri_row(int e) {
  int i = 0;
  while ((i + 1) * (i + 2) / 2 <= e) ++i;
  return i;
}
__host__ __device__ constexpr int tri_col(int e) { return e - tri_row(e) * (tri_row(e) + 1) / 2; }

// Reduce-scatter of N (<= 32) partial sums per lane across the 64 lanes of a
// wave: the two half-waves are added first, then on return lane l (and lane
// l + 32) holds the wave's sum of x[l % N].
template <int H, int N> __device__ __forceinline__ void rs_step(float (&x)[N], int l) {
  const bool up = (l & H) != 0;
#pragma unroll
  for (int e = 0; e < H; ++e) {
    const float send = up ? x[e] : x[e + H];
    const float keep = up ? x[e + H] : x[e];
    x[e] = keep + __shfl_xor(send, H);
  }
}
__device__ __forceinline__ float reduce_scatter32(float (&x)[32]) {
  const int l = lane_id();
#pragma unroll
  for (int e = 0; e < 32; ++e) x[e] += __shfl_xor(x[e], 32);
  rs_step<16>(x, l);
  rs_step<8>(x, l);
  rs_step<4>(x, l);
  rs_step<2>(x, l);
  rs_step<1>(x, l);
  return x[0];
}

__device__ __forceinline__ float allreduce64(float x) {
#pragma unroll
  for (int h = 32; h >= 1; h >>= 1) x += __shfl_xor(x, h);
  return x;
}

// Pair index of the non-adjacent block pairs (I, J), J <= I - 2, for C <= 64.
__device__ __forceinline__ int pair_index(int I, int J) { return I == 2 ? 0 : (J == 0 ? 1 : 2); }

// FPL consecutive elements as one aligned vector access.
template <typename T, int N> struct alignas(sizeof(T) * N) VecN { T e[N]; };
template <typename T, int N> __device__ __forceinline__ void ldvec(const T *p, bool ok, float (&o)[N]) {
  VecN<T, N> v;
  if (ok) v = *(const VecN<T, N> *)p;
#pragma unroll
  for (int i = 0; i < N; ++i) o[i] = ok ? (float)v.e[i] : 0.f;
}
template <typename T, int N> __device__ __forceinline__ void stvec(T *p, const float (&x)[N]) {
  VecN<T, N> v;
#pragma unroll
  for (int i = 0; i < N; ++i) v.e[i] = cvt<T>(x[i]);
  *(VecN<T, N> *)p = v;
}

// FPL consecutive elements as one buffer load / store of FPL * sizeof(T)
// bytes, kept as raw 32-bit words (out-of-range offsets read zero / drop).
template <typename T, int FPL>
__device__ __forceinline__ void ldraw(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint32_t (&r)[(FPL * sizeof(T) + 3) / 4]) {
  constexpr int B = FPL * sizeof(T);
  if constexpr (B == 2) {
    r[0] = __builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
  } else if constexpr (B == 4) {
    r[0] = __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
  } else if constexpr (B == 8) {
    const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
    r[0] = v[0];
    r[1] = v[1];
  } else {
    const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = v[i];
  }
}
template <typename T, int FPL>
__device__ __forceinline__ void unpack(const uint32_t (&r)[(FPL * sizeof(T) + 3) / 4], float (&o)[FPL]) {
#pragma unroll
  for (int i = 0; i < FPL; ++i) {
    if constexpr (sizeof(T) == 2) o[i] = __builtin_bit_cast(float, (r[i / 2] >> (16 * (i % 2))) << 16);
    else o[i] = __builtin_bit_cast(float, r[i]);
  }
}
template <typename T, int FPL>
__device__ __forceinline__ void straw(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float (&x)[FPL]) {
  constexpr int B = FPL * sizeof(T);
  VecN<T, FPL> v;
#pragma unroll
  for (int i = 0; i < FPL; ++i) v.e[i] = cvt<T>(x[i]);
  if constexpr (B == 2) {
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), rs, off, 0, 0);
  } else if constexpr (B == 4) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rs, off, 0, 0);
  } else if constexpr (B == 8) {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), rs, off, 0, 0);
  } else {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off, 0, 0);
  }
}

// PRE: the gate argument is the pre-activation of the gate epilogue.
template <typename T, int FPL, bool PRE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) prep_kernel(PrepArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int n = blockIdx.x, bh = blockIdx.y;
  const int w = wave_id(), l = lane_id(), g = l >> 4, j16 = l & 15;
  const int C = a.C, K = a.K, Kp = a.Kp, nb = C >> 4, ldk = a.ldk;
  const int t0 = n * C;
  const int rv = min(C, a.T - t0);
  const int64_t base = ((int64_t)bh * a.T + t0) * K;
  T *sQh = (T *)smem;
  T *sKs = sQh + C * ldk;
  float *sTot = (float *)(sKs + C * ldk);  // [nb][Kp] per-block sums of log alpha
  float *sG = sTot + 4 * Kp;              // [3][Kp] exp(sum of tot strictly between I and J)

  const T *q = (const T *)a.q + base, *k = (const T *)a.k + base;
  const T *la = (const T *)a.la + (a.sg ? (int64_t)bh * a.T + t0 : base);
  T *Qt = (T *)a.Qt + base, *Kt = (T *)a.Kt + base;
  T *Pg = (T *)a.P + ((int64_t)bh * a.N + n) * C * C;
  // lane l owns the FPL consecutive features k0 .. k0 + FPL - 1
  const int k0 = FPL * l;
  const bool fv = k0 < K;     // K is a multiple of 16, so all FPL are valid together
  const bool fp = k0 < Kp;    // inside the zero-padded LDS tiles

  // 0. every input row of this wave's block is requested at once (buffer
  // loads: rows past the sequence end and absent features read zero).
  constexpr int NW = (FPL * (int)sizeof(T) + 3) / 4;
  const int esz = sizeof(T);
  const uint32_t bytes = rsrc_bytes((int64_t)(a.T - t0) * K * esz);
  // an absent gate (alpha = 1) reads as log alpha = 0 from an empty range
  const uint32_t la_bytes = a.sg ? rsrc_bytes((int64_t)(a.T - t0) * esz) : bytes;
  const auto rs_la = make_rsrc(a.la ? la : q, a.la ? la_bytes : 0u), rs_q = make_rsrc(q, bytes), rs_k = make_rsrc(k, bytes);
  const uint32_t lane_off = fv ? (uint32_t)((16 * w * K + k0) * esz) : 0x80000000u;
  const uint32_t row_step = (uint32_t)(K * esz);
  uint32_t rla[16][NW], rq[16][NW], rk[16][NW];
  if (a.sg) {
    // scalar gate: the row's one value, broadcast to the features when unpacked
    const uint32_t o1 = fv ? (uint32_t)(16 * w * esz) : 0x80000000u;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (sizeof(T) == 2) rla[r][0] = __builtin_amdgcn_raw_buffer_load_b16(rs_la, o1 + r * esz, 0, 0);
      else rla[r][0] = __builtin_amdgcn_raw_buffer_load_b32(rs_la, o1 + r * esz, 0, 0);
    }
  } else {
#pragma unroll
    for (int r = 0; r < 16; ++r) ldraw<T, FPL>(rs_la, lane_off + r * row_step, rla[r]);
  }
  auto unpack_la = [&](int r, float (&x)[FPL]) {
    if (a.sg) {
      const float e = sizeof(T) == 2 ? __builtin_bit_cast(float, (rla[r][0] & 0xFFFFu) << 16)
                                     : __builtin_bit_cast(float, rla[r][0]);
#pragma unroll
      for (int f = 0; f < FPL; ++f) x[f] = e;
    } else {
      unpack<T, FPL>(rla[r], x);
    }
  };
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    ldraw<T, FPL>(rs_q, lane_off + r * row_step, rq[r]);
    ldraw<T, FPL>(rs_k, lane_off + r * row_step, rk[r]);
  }

  // 1. block sums of log alpha (with the gate epilogue, log alpha is formed
  // once here and kept for step 2).
  float tot[FPL], lav[PRE ? 16 : 1][FPL];
  {
#pragma unroll
    for (int f = 0; f < FPL; ++f) tot[f] = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float x[FPL];
      unpack_la(r, x);
#pragma unroll
      for (int f = 0; f < FPL; ++f) {
        if constexpr (PRE) {
          lav[r][f] = gate_la(x[f], a.inv_tau, fv && 16 * w + r < rv);
          tot[f] += lav[r][f];
        } else {
          tot[f] += x[f];
        }
      }
    }
#pragma unroll
    for (int f = 0; f < FPL; ++f)
      if (fp) sTot[w * Kp + k0 + f] = tot[f];
  }
  __syncthreads();

  float pre[FPL], Bl[FPL];
#pragma unroll
  for (int f = 0; f < FPL; ++f) {
    const int kf = k0 + f;
    pre[f] = 0.f;
    Bl[f] = 0.f;
    if (fp) {
      for (int w2 = 0; w2 < nb; ++w2) {
        const float t = sTot[w2 * Kp + kf];
        if (w2 < w) pre[f] += t;
        Bl[f] += t;
      }
      if (w == 2) sG[0 * Kp + kf] = __expf(sTot[1 * Kp + kf]);
      if (w == 3) {
        sG[1 * Kp + kf] = __expf(sTot[1 * Kp + kf] + sTot[2 * Kp + kf]);
        sG[2 * Kp + kf] = __expf(sTot[2 * Kp + kf]);
      }
    }
  }

  // 2. gated operands, from the block-local inclusive cumsum Bloc (kept, in
  // units of log2, for the diagonal block of step 4).
  float ez[FPL], ekt[FPL];
#pragma unroll
  for (int f = 0; f < FPL; ++f) {
    ez[f] = __expf(pre[f]);                    // b_{block start} / b_{chunk start}
    ekt[f] = __expf(Bl[f] - pre[f] - tot[f]);  // b_{chunk end} / b_{block end}
  }
  const auto rs_Qt = make_rsrc(Qt, bytes), rs_Kt = make_rsrc(Kt, bytes);
  float c[FPL], B2[16][FPL];
#pragma unroll
  for (int f = 0; f < FPL; ++f) c[f] = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = 16 * w + r;
    float xl[FPL], qv[FPL], kv[FPL], o1[FPL], o2[FPL], o3[FPL], o4[FPL];
    unpack_la(r, xl);
    unpack<T, FPL>(rq[r], qv);
    unpack<T, FPL>(rk[r], kv);
#pragma unroll
    for (int f = 0; f < FPL; ++f) {
      if constexpr (PRE) c[f] += lav[r][f];
      else c[f] += xl[f];
      B2[r][f] = c[f] * kLog2e;
      const float qhv = qv[f] * __expf(c[f]);           // <= |q|
      const float ksv = kv[f] * __expf(tot[f] - c[f]);  // <= |k|
      o1[f] = qhv * ez[f];
      o2[f] = ksv * ekt[f];
      o3[f] = qhv;
      o4[f] = ksv;
    }
    straw<T, FPL>(rs_Qt, lane_off + r * row_step, o1);
    straw<T, FPL>(rs_Kt, lane_off + r * row_step, o2);
    if (fp) {
      stvec<T, FPL>(sQh + row * ldk + k0, o3);
      stvec<T, FPL>(sKs + row * ldk + k0, o4);
    }
  }
  if (w == 0 && fv) {
    float gv[FPL];
#pragma unroll
    for (int f = 0; f < FPL; ++f) gv[f] = __expf(Bl[f]);
    float *gp = a.gam + ((int64_t)bh * a.N + n) * K + k0;
#pragma unroll
    for (int f = 0; f < FPL; ++f) gp[f] = gv[f];
  }

  // zeros: strict upper triangle of the diagonal block and every block J > w
  const int d0 = 16 * w;
  {
    const int i = l >> 2;
#pragma unroll
    for (int c4 = 0; c4 < 4; ++c4) {
      const int jj = 4 * (l & 3) + c4;
      if (jj > i) Pg[(d0 + i) * C + d0 + jj] = cvt<T>(0.f);
    }
    for (int idx = l; idx < 16 * (C - d0 - 16); idx += 64) {
      const int rr = idx / (C - d0 - 16), cc = idx - rr * (C - d0 - 16);
      Pg[(d0 + rr) * C + d0 + 16 + cc] = cvt<T>(0.f);
    }
  }
  __syncthreads();

  // 3. blocks (w, J < w) below the diagonal on the matrix cores.
  for (int J = 0; J < w; ++J) {
    f4 acc = zero4();
    for (int s = 0; s < Kp / 32; ++s) {
      frag_t<T> af = ld_row(sQh, ldk, d0, 32 * s);
      frag_t<T> bf = ld_row(sKs, ldk, 16 * J, 32 * s);
      if (J <= w - 2) {
        const float *gp = sG + pair_index(w, J) * Kp + 32 * s + 8 * g;
#pragma unroll
        for (int i = 0; i < 8; ++i) af[i] = cvt<T>((float)af[i] * gp[i]);
      }
      acc = mma<T>(acc, af, bf);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) Pg[(d0 + 4 * g + r) * C + 16 * J + j16] = cvt<T>(acc[r]);
  }

  // 4. the diagonal block in fp32 log space (Eq. 4): pair p = (i, j), j <= i,
  // of the block's 136 is sum_k q_ik k_jk 2^(B2_ik - B2_jk); each lane sums
  // its own features for 32 pairs at a time, then the wave reduces (pairs
  // 0..127 by reduce-scatter, lane l ending with pair p0 + l % 32; pairs
  // 128..135 by all-reduce).  The q, k values are the io-dtype inputs
  // themselves.
  auto pink = [&](auto p0, auto np, float (&x)[32]) {
    constexpr int P0 = decltype(p0)::value, NP = decltype(np)::value;
#pragma unroll
    for (int e = 0; e < NP; ++e) x[e] = 0.f;
#pragma unroll
    for (int f = 0; f < FPL; ++f) {
      float qf[16], kf[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float t[FPL];
        unpack<T, FPL>(rq[r], t);
        qf[r] = t[f];
        unpack<T, FPL>(rk[r], t);
        kf[r] = t[f];
      }
#pragma unroll
      for (int e = 0; e < NP; ++e) {
        const int i = tri_row(P0 + e), jj = tri_col(P0 + e);
        x[e] += qf[i] * kf[jj] * exp2f_fast(B2[i][f] - B2[jj][f]);
      }
    }
  };
  auto pink32 = [&](auto p0) {
    constexpr int P0 = decltype(p0)::value;
    float x[32];
    pink(p0, std::integral_constant<int, 32>{}, x);
    const float r = reduce_scatter32(x);
    if (l < 32) Pg[(d0 + tri_row(P0 + l)) * C + d0 + tri_col(P0 + l)] = cvt<T>(r);
  };
  pink32(std::integral_constant<int, 0>{});
  pink32(std::integral_constant<int, 32>{});
  pink32(std::integral_constant<int, 64>{});
  pink32(std::integral_constant<int, 96>{});
  {
    float x[32];
    pink(std::integral_constant<int, 128>{}, std::integral_constant<int, 8>{}, x);
    float rt = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float s = allreduce64(x[e]);
      if (l == e) rt = s;
    }
    if (l < 8) Pg[(d0 + 15) * C + d0 + 8 + l] = cvt<T>(rt);
  }
}

// Scalar gates (Table 1's scalar rows, alpha_t = gamma_t 1) and the absent
// gate (alpha = 1): the decay no longer depends on the feature, so with c the
// chunk-local inclusive cumsum of log gamma (one value per step)
//   Qt = q exp(c),  Kt = k exp(c_last - c),  gamma = exp(c_last) 1,
//   P = (q k^T) (.) D,  D_ij = exp(c_i - c_j) for j <= i, else 0,
// i.e. every block of P, the diagonal ones included, is a plain fp32-accumulated
// matrix-core product of the io-dtype inputs scaled by one fp32 exponential
// per entry -- no factorised operands, no block normalisers, no per-feature
// exponentials.  NG (no gate): c = 0, so D is the causal mask, gamma = 1, and
// Qt, Kt equal q, k: they are not written (the caller passes q and k in their
// place to the kernels that read them).
template <typename T, int FPL, bool PRE, bool NG>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) prep_plain_kernel(PrepArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int n = blockIdx.x, bh = blockIdx.y;
  const int w = wave_id(), l = lane_id(), g = l >> 4, j16 = l & 15;
  const int C = a.C, K = a.K, Kp = a.Kp, ldk = a.ldk;
  const int t0 = n * C;
  const int rv = min(C, a.T - t0);
  const int64_t base = ((int64_t)bh * a.T + t0) * K;
  T *sQ = (T *)smem;
  T *sK = sQ + C * ldk;
  const T *q = (const T *)a.q + base, *k = (const T *)a.k + base;
  T *Qt = (T *)a.Qt + base, *Kt = (T *)a.Kt + base;
  T *Pg = (T *)a.P + ((int64_t)bh * a.N + n) * C * C;
  const int k0 = FPL * l;
  const bool fv = k0 < K, fp = k0 < Kp;
  constexpr int NW = (FPL * (int)sizeof(T) + 3) / 4;
  const int esz = sizeof(T);
  const uint32_t bytes = rsrc_bytes((int64_t)(a.T - t0) * K * esz);
  const auto rs_q = make_rsrc(q, bytes), rs_k = make_rsrc(k, bytes);
  const uint32_t lane_off = fv ? (uint32_t)((16 * w * K + k0) * esz) : 0x80000000u;
  const uint32_t row_step = (uint32_t)(K * esz);
  uint32_t rq[16][NW], rk[16][NW];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    ldraw<T, FPL>(rs_q, lane_off + r * row_step, rq[r]);
    ldraw<T, FPL>(rs_k, lane_off + r * row_step, rk[r]);
  }

  // chunk-local inclusive cumsum of log gamma, in units of log2: lane t holds
  // step t's (every wave forms the whole chunk's; steps past the sequence end
  // or the chunk contribute 0)
  float c2 = 0.f;
  if constexpr (!NG) {
    const T *la = (const T *)a.la + (int64_t)bh * a.T + t0;
    const auto rs_la = make_rsrc(la, rsrc_bytes((int64_t)(a.T - t0) * esz));
    uint32_t raw;
    const uint32_t o1 = l < C ? (uint32_t)(l * esz) : 0x80000000u;
    if constexpr (sizeof(T) == 2) raw = __builtin_amdgcn_raw_buffer_load_b16(rs_la, o1, 0, 0) << 16;
    else raw = __builtin_amdgcn_raw_buffer_load_b32(rs_la, o1, 0, 0);
    float x = __builtin_bit_cast(float, raw);
    if constexpr (PRE) x = gate_la(x, a.inv_tau, l < rv);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float y = __shfl_up(x, o);
      if (l >= o) x += y;
    }
    c2 = x * kLog2e;
  }
  const float clast2 = NG ? 0.f : __shfl(c2, C - 1);

  // gated operands (scalar gates only), and the raw inputs into LDS
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = 16 * w + r;
    if constexpr (!NG) {
      const float cr = __shfl(c2, row);
      const float eq = exp2f_fast(cr), ek = exp2f_fast(clast2 - cr);
      float qv[FPL], kv[FPL], o1[FPL], o2[FPL];
      unpack<T, FPL>(rq[r], qv);
      unpack<T, FPL>(rk[r], kv);
#pragma unroll
      for (int f = 0; f < FPL; ++f) {
        o1[f] = qv[f] * eq;
        o2[f] = kv[f] * ek;
      }
      straw<T, FPL>(make_rsrc(Qt, bytes), lane_off + r * row_step, o1);
      straw<T, FPL>(make_rsrc(Kt, bytes), lane_off + r * row_step, o2);
    }
    if (fp) {
      float qv[FPL], kv[FPL];  // (exact round trip to the io dtype)
      unpack<T, FPL>(rq[r], qv);
      unpack<T, FPL>(rk[r], kv);
      stvec<T, FPL>(sQ + row * ldk + k0, qv);
      stvec<T, FPL>(sK + row * ldk + k0, kv);
    }
  }
  if (w == 0) {
    const float gv = exp2f_fast(clast2);
    float *gp = a.gam + ((int64_t)bh * a.N + n) * K;
    for (int kk = l; kk < K; kk += 64) gp[kk] = gv;
  }

  // zeros: every block J > w
  const int d0 = 16 * w;
  for (int idx = l; idx < 16 * (C - d0 - 16); idx += 64) {
    const int rr = idx / (C - d0 - 16), cc = idx - rr * (C - d0 - 16);
    Pg[(d0 + rr) * C + d0 + 16 + cc] = cvt<T>(0.f);
  }
  __syncthreads();

  // blocks (w, J <= w): q k^T on the matrix cores, then D
  float cr2[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) cr2[r] = NG ? 0.f : __shfl(c2, d0 + 4 * g + r);
  for (int J = 0; J <= w; ++J) {
    f4 acc = zero4();
    for (int s = 0; s < Kp / 32; ++s)
      acc = mma<T>(acc, ld_row(sQ, ldk, d0, 32 * s), ld_row(sK, ldk, 16 * J, 32 * s));
    const int col = 16 * J + j16;
    const float cc2 = NG ? 0.f : __shfl(c2, col);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = d0 + 4 * g + r;
      float v = 0.f;
      if (col <= row) v = NG ? acc[r] : acc[r] * exp2f_fast(cr2[r] - cc2);
      Pg[row * C + col] = cvt<T>(v);
    }
  }
}

static int round_up(int x, int m) { return (x + m - 1) / m * m; }

size_t lds_prep(const Shape &s) {
  const int Kp = round_up(s.K, 32), ldk = Kp + 32 / s.esz();
  return (size_t)2 * s.C * ldk * s.esz() + (size_t)7 * Kp * sizeof(float);
}

template <typename T, int FPL, bool PRE>
static hipError_t launch_prep_pre(const Shape &s, const PrepArgs &a, size_t lds, hipStream_t st) {
  // once per instantiation (thread-safe static initialisation), at the
  // maximum, since the LDS size depends on the shape
  static const hipError_t attr = hipFuncSetAttribute((const void *)prep_kernel<T, FPL, PRE>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  dim3 grid(s.N, s.BH), block(64 * (s.C / 16));
  hipLaunchKernelGGL((prep_kernel<T, FPL, PRE>), grid, block, lds, st, a);
  return hipGetLastError();
}

template <typename T, int FPL, bool PRE, bool NG>
static hipError_t launch_prep_plain(const Shape &s, const PrepArgs &a, size_t lds, hipStream_t st) {
  static const hipError_t attr = hipFuncSetAttribute((const void *)prep_plain_kernel<T, FPL, PRE, NG>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  dim3 grid(s.N, s.BH), block(64 * (s.C / 16));
  hipLaunchKernelGGL((prep_plain_kernel<T, FPL, PRE, NG>), grid, block, lds, st, a);
  return hipGetLastError();
}

template <typename T, int FPL>
static hipError_t launch_prep_t(const Shape &s, const PrepArgs &a, size_t lds, hipStream_t st) {
  if (!a.la) return launch_prep_plain<T, FPL, false, true>(s, a, lds, st);
  if (a.sg)
    return a.inv_tau != 0.f ? launch_prep_plain<T, FPL, true, false>(s, a, lds, st)
                            : launch_prep_plain<T, FPL, false, false>(s, a, lds, st);
  return a.inv_tau != 0.f ? launch_prep_pre<T, FPL, true>(s, a, lds, st)
                          : launch_prep_pre<T, FPL, false>(s, a, lds, st);
}

hipError_t launch_prep(const Shape &s, const void *q, const void *k, const void *la,
                       const Work &w, hipStream_t st) {
  PrepArgs a;
  a.q = q; a.k = k; a.la = la;
  a.Qt = w.Qt; a.Kt = w.Kt; a.P = w.P; a.gam = w.gam;
  a.T = s.T; a.K = s.K; a.Kp = round_up(s.K, 32); a.C = s.C; a.N = s.N;
  a.inv_tau = s.inv_tau;
  a.sg = s.sgate ? 1 : 0;
  a.ldk = a.Kp + 32 / s.esz();
  const size_t lds = lds_prep(s);
  const int fpl = (s.K + 63) / 64;
  if (s.io == IO_BF16) {
    if (fpl == 1) return launch_prep_t<bf16, 1>(s, a, lds, st);
    if (fpl == 2) return launch_prep_t<bf16, 2>(s, a, lds, st);
    return launch_prep_t<bf16, 4>(s, a, lds, st);
  }
  if (fpl == 1) return launch_prep_t<float, 1>(s, a, lds, st);
  if (fpl == 2) return launch_prep_t<float, 2>(s, a, lds, st);
  return launch_prep_t<float, 4>(s, a, lds, st);
}

}  // namespace gla
