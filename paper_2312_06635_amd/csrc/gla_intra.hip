// gla_intra.hip -- the intra-chunk part of the backward (App. B, Alg. 4/6 as
// corrected in the header of gla_vsweep.hip), chunk-parallel: none of it
// depends on the states, so it is computed once per (head, chunk) here and
// the key sweeps keep only the state recurrences.
//
// Per chunk (rows t of the chunk, B = chunk-local inclusive cumsum of log
// alpha, dP = (dO V^T) (.) M):
//   dq_intra[i] = sum_{j <= i} dP_ij k_j (.) exp(B_i - B_j)
//   dk_intra[j] = sum_{i >= j} dP_ij q_i (.) exp(B_i - B_j)
//   dA_intra[t] = q_t (.) dq_intra[t] - k_t (.) dk_intra[t]   (Sec. 4.3)
// It runs between the key sweeps: it writes dq = dq_inter + dq_intra (the dq
// sweep's fp32 dq_inter in), and for the dk sweep dk_intra, the in-chunk
// reverse cumsum of dA_intra (io dtype: each is added once to an fp32
// inter-chunk term) and the chunk total of dA_intra (fp32: the gate gradient
// carries it across chunks).  dP comes from the dq sweep, which streams V and
// dO anyway.
//
// One workgroup per (chunk, head), wave w = the 16-row block w of the chunk.
//   1. The chunk's dP (fp32, masked, stored transposed) into LDS.
//   2. For each group of 64 key features (lane = feature):
//      - gate cumsums of the wave's block; the sub-chunk ("pink") diagonal
//        block in fp32 log space on the vector ALUs: one exponential
//        2^(B2_i - B2_j) per pair, shared by the dq and dk sums;
//      - the blocks between sub-chunks ("orange") on the matrix cores: with
//        normalisers at block boundaries every exponent is <= 0,
//          dq_I = exp(Bloc_I) (.) sum_{J<I} g_IJ (.) dP_IJ (k_J (.) exp(tot_J - Bloc_J))
//          dk_J = exp(tot_J - Bloc_J) (.) sum_{I>J} g_IJ (.) dP_IJ^T (q_I (.) exp(Bloc_I))
//        (Bloc = block-local cumsum, tot = block total, g_IJ = decay of the
//        blocks strictly between J and I), the fp32 operands split into bf16
//        hi + lo (three products) so that the gate gradient keeps fp32
//        accuracy;
//      - per (row, feature): the two parts added, dA formed and summed
//        backwards over the chunk.
#include <type_traits>

#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

struct IntraArgs {
  const void *q, *k, *la;
  const float *dP;        // [BH][N][C][C] fp32, transposed ([s][t])
  const float *dqr;       // [BH][T][K] fp32 dq_inter
  void *dq;               // [BH][T][K] io: the layer's dq
  void *dki, *dai;        // [BH][T][K] io
  float *dat;             // [BH][N][K] fp32
  int T, K, C, N;
  int sg;         // scalar gate: la is [BH][T]
  int ng;         // no gate and no gate gradient
  float inv_tau;  // gate epilogue (0: la holds log alpha)
};

template <typename T> __device__ __forceinline__ uint32_t ld_el(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
  if constexpr (sizeof(T) == 2) return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
  else return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
}
template <typename T> __device__ __forceinline__ float el_f(uint32_t raw) {
  if constexpr (sizeof(T) == 2) return __builtin_bit_cast(float, raw << 16);
  else return __builtin_bit_cast(float, raw);
}
template <typename T> __device__ __forceinline__ void st_el(__amdgpu_buffer_rsrc_t rs, uint32_t off, float x) {
  if constexpr (sizeof(T) == 2)
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, cvt<bf16>(x)), rs, off, 0, 0);
  else
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), rs, off, 0, 0);
}

// acc += a b for fp32 operands: on the bf16 path both are split into hi + lo
// and the three significant cross products accumulated.
template <typename T> __device__ __forceinline__ f4 mma3(f4 acc, const f8 &a, const f8 &b) {
  if constexpr (sizeof(T) == 2) {
    frag_t<T> ah, al, bh, bl;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ah[i] = cvt<T>(a[i]);
      al[i] = cvt<T>(a[i] - (float)ah[i]);
      bh[i] = cvt<T>(b[i]);
      bl[i] = cvt<T>(b[i] - (float)bh[i]);
    }
    acc = mma<T>(acc, ah, bh);
    acc = mma<T>(acc, ah, bl);
    return mma<T>(acc, al, bh);
  } else {
    return mma<T>(acc, a, b);
  }
}

// An fp32 operand of mma3, split once when it is reused: bf16 hi + lo (the
// fp32 path keeps the value itself in hi).
template <typename T> struct Split {
  frag_t<T> hi, lo;
};
template <typename T> __device__ __forceinline__ Split<T> split8(const f8 &a) {
  Split<T> r;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      r.hi[i] = cvt<T>(a[i]);
      r.lo[i] = cvt<T>(a[i] - (float)r.hi[i]);
    }
  } else {
    r.hi = a;
  }
  return r;
}
// mma3 with the first operand already split.
template <typename T> __device__ __forceinline__ f4 mma3s(f4 acc, const Split<T> &a, const f8 &b) {
  if constexpr (sizeof(T) == 2) {
    frag_t<T> bh, bl;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      bh[i] = cvt<T>(b[i]);
      bl[i] = cvt<T>(b[i] - (float)bh[i]);
    }
    acc = mma<T>(acc, a.hi, bh);
    acc = mma<T>(acc, a.hi, bl);
    return mma<T>(acc, a.lo, bh);
  } else {
    return mma<T>(acc, a.hi, b);
  }
}

template <int C> struct IntraLayout {
  static constexpr int NB = C / 16;
  static constexpr int LDD = C + 4;   // dP rows; per-feature rows of the group tiles
  static constexpr int LDO = 17;      // per-wave result tiles [64 features][16 rows]
  static constexpr size_t offdP = 0;                                   // [C][LDD] fp32
  static constexpr size_t offTot = offdP + 4 * C * LDD;                // [NB][64] block sums of log alpha
  static constexpr size_t offTA = offTot + 4 * NB * 64;                // [NB][64] block sums of dA
  static constexpr size_t offQz = offTA + 4 * NB * 64;                 // [64][LDD] q (.) exp(Bloc)
  static constexpr size_t offKz = offQz + 4 * 64 * LDD;                // [64][LDD] k (.) exp(tot - Bloc)
  static constexpr size_t offO = offQz;                                // (aliased) [NB][2][64][LDO]
  static constexpr size_t total = offKz + 4 * 64 * LDD;
  static_assert(offO + 4 * NB * 2 * 64 * LDO <= total, "result tiles fit over the group tiles");
};

template <typename T, int C, bool PRE>
__global__ void __launch_bounds__(64 * (C / 16)) __attribute__((amdgpu_waves_per_eu(2))) intra_kernel(IntraArgs a) {
  using L = IntraLayout<C>;
  constexpr int NB = L::NB, LDD = L::LDD, LDO = L::LDO;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float *sdP = (float *)(smem + L::offdP);
  float *sTot = (float *)(smem + L::offTot), *sTA = (float *)(smem + L::offTA);
  float *sQz = (float *)(smem + L::offQz), *sKz = (float *)(smem + L::offKz);
  float *sO = (float *)(smem + L::offO);

  const int n = blockIdx.x, bh = blockIdx.y;
  const int w = wave_id(), l = lane_id(), g16 = l >> 4, j16 = l & 15;
  const int K = a.K, T_ = a.T;
  const int t0 = n * C, rv = min(C, T_ - t0);
  const int esz = sizeof(T);

  // ---- inputs of the feature groups (lane = feature): the group's rows of
  // q, k and the gate
  const int lrow = a.sg ? 1 : K;  // gate elements per step
  const T *qc = (const T *)a.q + ((int64_t)bh * T_ + t0) * K;
  const T *kc = (const T *)a.k + ((int64_t)bh * T_ + t0) * K;
  const uint32_t kbytes = rsrc_bytes((int64_t)(T_ - t0) * K * esz);
  const auto rs_q = make_rsrc(qc, kbytes), rs_k = make_rsrc(kc, kbytes);
  // an absent gate (alpha = 1) reads as log alpha = 0 from an empty range
  const auto rs_la = make_rsrc(a.la ? (const T *)a.la + ((int64_t)bh * T_ + t0) * lrow : qc,
                               a.la ? rsrc_bytes((int64_t)(T_ - t0) * lrow * esz) : 0u);
  const auto rs_dq = make_rsrc((T *)a.dq + ((int64_t)bh * T_ + t0) * K, kbytes);
  const auto rs_dki = make_rsrc((T *)a.dki + ((int64_t)bh * T_ + t0) * K, kbytes);
  const auto rs_dai = make_rsrc((T *)a.dai + ((int64_t)bh * T_ + t0) * K, kbytes);
  float *datc = a.dat + ((int64_t)bh * a.N + n) * K;
  const int NG = (K + 63) / 64;

  const auto rs_dqr = make_rsrc(a.dqr + ((int64_t)bh * T_ + t0) * K, rsrc_bytes((int64_t)(T_ - t0) * K * 4));
  uint32_t nq[16], nk[16], nl[16];
  auto issue_group = [&](int gi) {
    const int f = 64 * gi + l;
    const bool fv = f < K;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 16 * w + r;
      const uint32_t off = fv ? (uint32_t)((row * K + f) * esz) : 0x80000000u;
      nq[r] = ld_el<T>(rs_q, off);
      nk[r] = ld_el<T>(rs_k, off);
      nl[r] = ld_el<T>(rs_la, a.sg ? (fv ? (uint32_t)(row * esz) : 0x80000000u) : off);
    }
  };

  // ---- 1. the chunk's dP, transposed back into rows (thread: C/4
  // consecutive t of one s)
  {
    constexpr int PER = C / 4;  // floats per thread: C * C over 64 NB = 4 C threads
    const int e0 = (int)threadIdx.x * PER, sc = e0 / C, tb = e0 % C;
    const float *src = a.dP + ((int64_t)bh * a.N + n) * C * C + e0;
#pragma unroll
    for (int u = 0; u < PER; u += 4) {
      const f4 x = *(const f4 *)(src + u);
#pragma unroll
      for (int r = 0; r < 4; ++r) sdP[(tb + u + r) * LDD + sc] = x[r];
    }
  }

  __syncthreads();  // the chunk's dP rows are complete

  // ---- 2. feature groups
  for (int gi = 0; gi < NG; ++gi) {
    const int f = 64 * gi + l;
    const bool fv = f < K;
    // the block's rows of q, k and the gate, for this lane's feature
    uint32_t rq[16], rk[16], rl[16], rr[16];
    issue_group(gi);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      rq[r] = nq[r];
      rk[r] = nk[r];
      rl[r] = nl[r];
    }
    // dq_inter of this group's rows: needed only at the combine
#pragma unroll
    for (int r = 0; r < 16; ++r)
      rr[r] = __builtin_amdgcn_raw_buffer_load_b32(rs_dqr, fv ? (uint32_t)(((16 * w + r) * K + f) * 4) : 0x80000000u, 0, 0);
    float q[16], kk[16], c[16];
    float run = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float x = el_f<T>(rl[r]);
      if constexpr (PRE) x = gate_la(x, a.inv_tau, fv && 16 * w + r < rv);
      run += x;
      c[r] = run;  // Bloc
      q[r] = el_f<T>(rq[r]);
      kk[r] = el_f<T>(rk[r]);
    }
    const float tot = run;
    // (block sums and group tiles are read after B2; the previous group's
    // result tiles, which the group tiles overlay, were consumed before its B4)
    sTot[w * 64 + l] = tot;

    // operands of the orange blocks, feature-major
#pragma unroll
    for (int r = 0; r < 16; r += 4) {
      f4 qz, kz;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        qz[u] = q[r + u] * __expf(c[r + u]);
        kz[u] = kk[r + u] * __expf(tot - c[r + u]);
      }
      *(f4 *)(sQz + l * LDD + 16 * w + r) = qz;
      *(f4 *)(sKz + l * LDD + 16 * w + r) = kz;
    }

    // pink: the diagonal block in fp32 log space, one exponential per pair
    // shared by both sums (dP rows read as wave-uniform broadcasts)
    float dqp[16], dkp[16], c2[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dqp[r] = dkp[r] = 0.f;
      c2[r] = c[r] * kLog2e;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float *prow = sdP + (16 * w + i) * LDD + 16 * w;
      float p[16];
#pragma unroll
      for (int j4 = 0; j4 <= i / 4; ++j4) {
        const f4 v4 = *(const f4 *)(prow + 4 * j4);
#pragma unroll
        for (int u = 0; u < 4; ++u) p[4 * j4 + u] = v4[u];
      }
#pragma unroll
      for (int j = 0; j <= i; ++j) {
        const float t = p[j] * exp2f_fast(c2[i] - c2[j]);
        dqp[i] += t * kk[j];
        dkp[j] += t * q[i];
      }
    }
    // finish the sums here: sunk to their use after the orange blocks, the 136
    // exponentials would all stay live across them
#pragma unroll
    for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(dqp[r]), "+v"(dkp[r]));
    __syncthreads();  // B2: group tiles complete

    // orange on the matrix cores: wave w forms dq for row block I = w and dk
    // for column block J = w, four 16-feature tiles each.  The dP operands
    // (the same for every tile) are split once.
    constexpr int NSTEP = NB / 2 > 0 ? NB / 2 : 1;
    Split<T> aq[NSTEP], ak[NSTEP];
#pragma unroll
    for (int s = 0; s < NB / 2; ++s) {
      const float *ap = sdP + (16 * w + j16) * LDD + 32 * s + 8 * g16;
      const f4 a0 = *(const f4 *)ap, a1 = *(const f4 *)(ap + 4);
      aq[s] = split8<T>(f8{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]});
      f8 at;
#pragma unroll
      for (int u = 0; u < 8; ++u) at[u] = sdP[(32 * s + 8 * g16 + u) * LDD + 16 * w + j16];
      ak[s] = split8<T>(at);
    }
    f4 oq[4], ok[4];
#pragma unroll
    for (int ft = 0; ft < 4; ++ft) {
      // (one tile at a time: unbounded hoisting of the tiles' operand reads
      // would hold every fragment of all four tiles in registers)
      __builtin_amdgcn_sched_barrier(0);
      oq[ft] = ok[ft] = zero4();
      const int fl = 16 * ft + j16;  // feature of this lane's output column (group-local)
      // dq: sum over J < w of dP_wJ (kz_J g_wJ)
#pragma unroll
      for (int s = 0; s < NB / 2; ++s) {
        if (32 * s >= 16 * w) continue;  // both blocks at or right of the diagonal
        const int J = 2 * s + (g16 >> 1);
        float lg = 0.f;
#pragma unroll
        for (int b = 0; b < NB; ++b)
          if (b > J && b < w) lg += sTot[b * 64 + fl];
        const float sc = J < w ? __expf(lg) : 0.f;
        const float *bp = sKz + fl * LDD + 32 * s + 8 * g16;
        const f4 b0 = *(const f4 *)bp, b1 = *(const f4 *)(bp + 4);
        const f8 bf = f8{b0[0] * sc, b0[1] * sc, b0[2] * sc, b0[3] * sc, b1[0] * sc, b1[1] * sc, b1[2] * sc, b1[3] * sc};
        oq[ft] = mma3s<T>(oq[ft], aq[s], bf);
      }
      // dk: sum over I > w of dP_Iw^T (qz_I g_Iw)
#pragma unroll
      for (int s = 0; s < NB / 2; ++s) {
        if (32 * s + 31 < 16 * (w + 1)) continue;  // both blocks at or above the diagonal
        const int I = 2 * s + (g16 >> 1);
        float lg = 0.f;
#pragma unroll
        for (int b = 0; b < NB; ++b)
          if (b > w && b < I) lg += sTot[b * 64 + fl];
        const float sc = I > w ? __expf(lg) : 0.f;
        const float *bp = sQz + fl * LDD + 32 * s + 8 * g16;
        const f4 b0 = *(const f4 *)bp, b1 = *(const f4 *)(bp + 4);
        const f8 bf = f8{b0[0] * sc, b0[1] * sc, b0[2] * sc, b0[3] * sc, b1[0] * sc, b1[1] * sc, b1[2] * sc, b1[3] * sc};
        ok[ft] = mma3s<T>(ok[ft], ak[s], bf);
      }
    }
    __syncthreads();  // B3: every wave is done with the group tiles, which the result tiles overlay

    float *oqw = sO + (w * 2 + 0) * 64 * LDO, *okw = sO + (w * 2 + 1) * 64 * LDO;
#pragma unroll
    for (int ft = 0; ft < 4; ++ft)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        oqw[(16 * ft + j16) * LDO + 4 * g16 + r] = oq[ft][r];
        okw[(16 * ft + j16) * LDO + 4 * g16 + r] = ok[ft][r];
      }
    // (the wave reads back only what it wrote: LDS keeps one wave's accesses in order)
    float dA[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 16 * w + r;
      const float dq = __expf(c[r]) * oqw[l * LDO + r] + dqp[r];
      const float dk = __expf(tot - c[r]) * okw[l * LDO + r] + dkp[r];
      const uint32_t off = fv ? (uint32_t)((row * K + f) * esz) : 0x80000000u;
      st_el<T>(rs_dq, off, __builtin_bit_cast(float, rr[r]) + dq);
      st_el<T>(rs_dki, off, dk);
      dA[r] = q[r] * dq - kk[r] * dk;
    }
    float sa = 0.f;
#pragma unroll
    for (int r = 15; r >= 0; --r) {
      sa += dA[r];
      dA[r] = sa;
    }
    sTA[w * 64 + l] = sa;
    __syncthreads();  // B4: block sums of dA published
    float later = 0.f;
#pragma unroll
    for (int b = 0; b < NB; ++b)
      if (b > w) later += sTA[b * 64 + l];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 16 * w + r;
      st_el<T>(rs_dai, fv ? (uint32_t)((row * K + f) * esz) : 0x80000000u, dA[r] + later);
    }
    if (w == 0 && fv) datc[f] = sa + later;
  }
}

// acc += a b with a split once and b exact in the io dtype (bf16: hi b + lo b).
template <typename T> __device__ __forceinline__ f4 mma2s(f4 acc, const Split<T> &a, const frag_t<T> &b) {
  acc = mma<T>(acc, a.hi, b);
  if constexpr (sizeof(T) == 2) acc = mma<T>(acc, a.lo, b);
  return acc;
}

// Scalar gates and the absent gate: the decay D_ij = exp(c_i - c_j) (c the
// chunk-local cumsum of log gamma; D = 1 without a gate) is shared by every
// feature, so with dPD = dP (.) D (.) M
//   dq_intra = dPD K,   dk_intra = dPD^T Q,
// each one matrix-core product per 16x16 output tile and 32-row slab: dPD is
// split into bf16 hi + lo once per chunk, q and k enter exactly (no
// factorised operands, no per-feature exponentials).  The gate gradient's
// parts (dai, dat) are formed as in the per-feature kernel; NG (no gate)
// skips them.
template <typename T, int C, bool PRE, bool NG>
__global__ void __launch_bounds__(64 * (C / 16)) __attribute__((amdgpu_waves_per_eu(2)))
intra_plain_kernel(IntraArgs a) {
  using L = IntraLayout<C>;
  constexpr int NB = L::NB, LDD = L::LDD, LDO = L::LDO;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float *sdP = (float *)(smem + L::offdP), *sTA = (float *)(smem + L::offTA);
  float *sQz = (float *)(smem + L::offQz), *sKz = (float *)(smem + L::offKz);
  float *sO = (float *)(smem + L::offO);

  const int n = blockIdx.x, bh = blockIdx.y;
  const int w = wave_id(), l = lane_id(), g16 = l >> 4, j16 = l & 15;
  const int K = a.K, T_ = a.T;
  const int t0 = n * C, rv = min(C, T_ - t0);
  const int esz = sizeof(T);
  const T *qc = (const T *)a.q + ((int64_t)bh * T_ + t0) * K;
  const T *kc = (const T *)a.k + ((int64_t)bh * T_ + t0) * K;
  const uint32_t kbytes = rsrc_bytes((int64_t)(T_ - t0) * K * esz);
  const auto rs_q = make_rsrc(qc, kbytes), rs_k = make_rsrc(kc, kbytes);
  const auto rs_dq = make_rsrc((T *)a.dq + ((int64_t)bh * T_ + t0) * K, kbytes);
  const auto rs_dki = make_rsrc((T *)a.dki + ((int64_t)bh * T_ + t0) * K, kbytes);
  const auto rs_dqr = make_rsrc(a.dqr + ((int64_t)bh * T_ + t0) * K, rsrc_bytes((int64_t)(T_ - t0) * K * 4));

  // chunk-local inclusive cumsum of log gamma in units of log2, lane t = step t
  float c2 = 0.f;
  if constexpr (!NG) {
    // (an absent gate whose gradient is wanted reads as log alpha = 0 from an
    // empty range; the per-feature dA below is then that gradient's share)
    const auto rs_la = make_rsrc(a.la ? (const T *)a.la + (int64_t)bh * T_ + t0 : qc,
                                 a.la ? rsrc_bytes((int64_t)(T_ - t0) * esz) : 0u);
    float x = el_f<T>(ld_el<T>(rs_la, l < C ? (uint32_t)(l * esz) : 0x80000000u));
    if constexpr (PRE) x = gate_la(x, a.inv_tau, l < rv);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float y = __shfl_up(x, o);
      if (l >= o) x += y;
    }
    c2 = x * kLog2e;
  }

  // ---- 1. dPD rows into LDS (thread: C/4 consecutive t of one s; dP is
  // stored transposed and already masked)
  {
    constexpr int PER = C / 4;
    const int e0 = (int)threadIdx.x * PER, sc = e0 / C, tb = e0 % C;
    const float *src = a.dP + ((int64_t)bh * a.N + n) * C * C + e0;
    const float cs = NG ? 0.f : __shfl(c2, sc);
#pragma unroll
    for (int u = 0; u < PER; u += 4) {
      const f4 x = *(const f4 *)(src + u);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = tb + u + r;
        float v = x[r];
        if constexpr (!NG) {
          // (the cross-lane read runs in every lane: a lane that skipped it
          // would hand its readers no value)
          const float ct = __shfl(c2, t);
          v = sc <= t ? v * exp2f_fast(ct - cs) : 0.f;
        }
        sdP[t * LDD + sc] = v;
      }
    }
  }
  __syncthreads();

  // the dPD operands of this wave's row block (dq) and column block (dk),
  // split once for every feature tile
  // (32-row slabs; with C = 16 the slots past the chunk are zeros)
  constexpr int NSB = (C + 31) / 32;
  const bool slot_in = C >= 32 || g16 < 2;
  Split<T> aq[NSB], ak[NSB];
#pragma unroll
  for (int s = 0; s < NSB; ++s) {
    f8 aw = f8{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, at = aw;
    if (slot_in) {
      const float *ap = sdP + (16 * w + j16) * LDD + 32 * s + 8 * g16;
      const f4 a0 = *(const f4 *)ap, a1 = *(const f4 *)(ap + 4);
      aw = f8{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
#pragma unroll
      for (int u = 0; u < 8; ++u) at[u] = sdP[(32 * s + 8 * g16 + u) * LDD + 16 * w + j16];
    }
    aq[s] = split8<T>(aw);
    ak[s] = split8<T>(at);
  }

  // ---- 2. feature groups (lane = feature)
  const int NGR = (K + 63) / 64;
  for (int gi = 0; gi < NGR; ++gi) {
    const int f = 64 * gi + l;
    const bool fv = f < K;
    uint32_t rq[16], rk[16], rr[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const uint32_t off = fv ? (uint32_t)(((16 * w + r) * K + f) * esz) : 0x80000000u;
      rq[r] = ld_el<T>(rs_q, off);
      rk[r] = ld_el<T>(rs_k, off);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r)
      rr[r] = __builtin_amdgcn_raw_buffer_load_b32(rs_dqr, fv ? (uint32_t)(((16 * w + r) * K + f) * 4) : 0x80000000u, 0, 0);
    float q[16], kk[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      q[r] = el_f<T>(rq[r]);
      kk[r] = el_f<T>(rk[r]);
    }
    // (the previous group's result tiles, which these overlay, were consumed
    // before its last barrier)
#pragma unroll
    for (int r = 0; r < 16; r += 4) {
      *(f4 *)(sQz + l * LDD + 16 * w + r) = f4{q[r], q[r + 1], q[r + 2], q[r + 3]};
      *(f4 *)(sKz + l * LDD + 16 * w + r) = f4{kk[r], kk[r + 1], kk[r + 2], kk[r + 3]};
    }
    __syncthreads();  // group tiles complete

    f4 oq[4], ok[4];
#pragma unroll
    for (int ft = 0; ft < 4; ++ft) {
      __builtin_amdgcn_sched_barrier(0);
      oq[ft] = ok[ft] = zero4();
      const int fl = 16 * ft + j16;
      // dq of row block w: slabs holding a block J <= w
#pragma unroll
      for (int s = 0; s < NSB; ++s) {
        if (32 * s > 16 * w + 15) continue;
        const float *bp = sKz + fl * LDD + 32 * s + 8 * g16;
        const f4 b0 = slot_in ? *(const f4 *)bp : zero4(), b1 = slot_in ? *(const f4 *)(bp + 4) : zero4();
        frag_t<T> bf;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          bf[u] = cvt<T>(b0[u]);
          bf[4 + u] = cvt<T>(b1[u]);
        }
        oq[ft] = mma2s<T>(oq[ft], aq[s], bf);
      }
      // dk of column block w: slabs holding a block I >= w
#pragma unroll
      for (int s = 0; s < NSB; ++s) {
        if (32 * s + 31 < 16 * w) continue;
        const float *bp = sQz + fl * LDD + 32 * s + 8 * g16;
        const f4 b0 = slot_in ? *(const f4 *)bp : zero4(), b1 = slot_in ? *(const f4 *)(bp + 4) : zero4();
        frag_t<T> bf;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          bf[u] = cvt<T>(b0[u]);
          bf[4 + u] = cvt<T>(b1[u]);
        }
        ok[ft] = mma2s<T>(ok[ft], ak[s], bf);
      }
    }
    __syncthreads();  // every wave is done with the group tiles, which the result tiles overlay

    float *oqw = sO + (w * 2 + 0) * 64 * LDO, *okw = sO + (w * 2 + 1) * 64 * LDO;
#pragma unroll
    for (int ft = 0; ft < 4; ++ft)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        oqw[(16 * ft + j16) * LDO + 4 * g16 + r] = oq[ft][r];
        okw[(16 * ft + j16) * LDO + 4 * g16 + r] = ok[ft][r];
      }
    // (the wave reads back only what it wrote: LDS keeps one wave's accesses in order)
    float dA[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 16 * w + r;
      const float dq = oqw[l * LDO + r], dk = okw[l * LDO + r];
      const uint32_t off = fv ? (uint32_t)((row * K + f) * esz) : 0x80000000u;
      st_el<T>(rs_dq, off, __builtin_bit_cast(float, rr[r]) + dq);
      st_el<T>(rs_dki, off, dk);
      dA[r] = q[r] * dq - kk[r] * dk;
    }
    if constexpr (!NG) {
      const auto rs_dai = make_rsrc((T *)a.dai + ((int64_t)bh * T_ + t0) * K, kbytes);
      float sa = 0.f;
#pragma unroll
      for (int r = 15; r >= 0; --r) {
        sa += dA[r];
        dA[r] = sa;
      }
      sTA[w * 64 + l] = sa;
      __syncthreads();  // block sums of dA published
      float later = 0.f;
#pragma unroll
      for (int b = 0; b < NB; ++b)
        if (b > w) later += sTA[b * 64 + l];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 16 * w + r;
        st_el<T>(rs_dai, fv ? (uint32_t)((row * K + f) * esz) : 0x80000000u, dA[r] + later);
      }
      if (w == 0 && fv) a.dat[((int64_t)bh * a.N + n) * K + f] = sa + later;
    } else {
      __syncthreads();  // result tiles consumed before the next group's tiles overlay them
    }
  }
}

template <typename T, int C, bool PRE>
hipError_t launch_intra_t(const Shape &s, const IntraArgs &a, hipStream_t st) {
  static const hipError_t attr = hipFuncSetAttribute((const void *)intra_kernel<T, C, PRE>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  hipLaunchKernelGGL((intra_kernel<T, C, PRE>), dim3(s.N, s.BH), dim3(64 * (C / 16)), IntraLayout<C>::total, st, a);
  return hipGetLastError();
}

template <typename T, int C, bool PRE, bool NG>
hipError_t launch_intra_plain(const Shape &s, const IntraArgs &a, hipStream_t st) {
  static const hipError_t attr = hipFuncSetAttribute((const void *)intra_plain_kernel<T, C, PRE, NG>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  hipLaunchKernelGGL((intra_plain_kernel<T, C, PRE, NG>), dim3(s.N, s.BH), dim3(64 * (C / 16)), IntraLayout<C>::total,
                     st, a);
  return hipGetLastError();
}

template <typename T, int C>
hipError_t launch_intra_c(const Shape &s, const IntraArgs &a, hipStream_t st) {
  if (a.ng) return launch_intra_plain<T, C, false, true>(s, a, st);
  if (a.sg || !a.la)
    return a.inv_tau != 0.f ? launch_intra_plain<T, C, true, false>(s, a, st)
                            : launch_intra_plain<T, C, false, false>(s, a, st);
  return a.inv_tau != 0.f ? launch_intra_t<T, C, true>(s, a, st) : launch_intra_t<T, C, false>(s, a, st);
}

template <typename T>
hipError_t launch_intra_io(const Shape &s, const IntraArgs &a, hipStream_t st) {
  if (s.C == 16) return launch_intra_c<T, 16>(s, a, st);
  if (s.C == 32) return launch_intra_c<T, 32>(s, a, st);
  return launch_intra_c<T, 64>(s, a, st);
}

}  // namespace

size_t lds_bwd_intra(const Shape &s) {
  return s.C == 16 ? IntraLayout<16>::total : (s.C == 32 ? IntraLayout<32>::total : IntraLayout<64>::total);
}

hipError_t launch_bwd_intra(const Shape &s, const void *q, const void *k, const void *la, void *dq, const Work &w,
                            hipStream_t st, bool ng) {
  IntraArgs a;
  a.q = q; a.k = k; a.la = la; a.dP = w.dP; a.dqr = w.dqr; a.dq = dq;
  a.dki = w.dki; a.dai = w.dai; a.dat = w.dat;
  a.T = s.T; a.K = s.K; a.C = s.C; a.N = s.N;
  a.sg = s.sgate ? 1 : 0;
  a.ng = ng ? 1 : 0;
  a.inv_tau = s.inv_tau;
  return s.io == IO_BF16 ? launch_intra_io<bf16>(s, a, st) : launch_intra_io<float>(s, a, st);
}

}  // namespace gla
