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
// and the chunk writes dq_intra, dk_intra, the in-chunk reverse cumsum of
// dA_intra (io dtype: each is added once to an fp32 inter-chunk term) and the
// chunk total of dA_intra (fp32: the gate gradient carries it across chunks).
//
// One workgroup per (chunk, head), wave w = the 16-row block w of the chunk.
//   1. dP: wave w forms the 16 x 16 blocks (w, J <= w) of dO V^T on the
//      matrix cores (bf16, fp32 accumulate; fp32 MFMA for fp32 io), operands
//      straight from memory, and stores its 16 rows (masked) to LDS.
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
  const void *q, *k, *la, *v, *dO;
  void *dqi, *dki, *dai;  // [BH][T][K] io
  float *dat;             // [BH][N][K] fp32
  int T, K, V, C, N;
  int sg;         // scalar gate: la is [BH][T]
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

// One fragment (8 consecutive elements of a row) straight from memory.
template <typename T> __device__ __forceinline__ frag_t<T> ld_frag(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
  if constexpr (sizeof(T) == 2) {
    return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
  } else {
    const f4 a = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
    const f4 b = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16, 0, 0));
    return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
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
__global__ void __launch_bounds__(64 * (C / 16)) intra_kernel(IntraArgs a) {
  using L = IntraLayout<C>;
  constexpr int NB = L::NB, LDD = L::LDD, LDO = L::LDO;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float *sdP = (float *)(smem + L::offdP);
  float *sTot = (float *)(smem + L::offTot), *sTA = (float *)(smem + L::offTA);
  float *sQz = (float *)(smem + L::offQz), *sKz = (float *)(smem + L::offKz);
  float *sO = (float *)(smem + L::offO);

  const int n = blockIdx.x, bh = blockIdx.y;
  const int w = wave_id(), l = lane_id(), g16 = l >> 4, j16 = l & 15;
  const int K = a.K, V = a.V, T_ = a.T;
  const int t0 = n * C, rv = min(C, T_ - t0);
  const int esz = sizeof(T);

  // ---- 1. dP rows of block w: blocks (w, J <= w) of dO V^T
  {
    const T *dOc = (const T *)a.dO + ((int64_t)bh * T_ + t0) * V;
    const T *vc = (const T *)a.v + ((int64_t)bh * T_ + t0) * V;
    const uint32_t vb = rsrc_bytes((int64_t)(T_ - t0) * V * esz);
    const auto rs_do = make_rsrc(dOc, vb), rs_v = make_rsrc(vc, vb);
    f4 acc[NB];
#pragma unroll
    for (int J = 0; J < NB; ++J) acc[J] = zero4();
    const uint32_t arow = (uint32_t)((16 * w + j16) * V) * esz;
#pragma unroll 2
    for (int s = 0; s < (V + 31) / 32; ++s) {
      const int col = 32 * s + 8 * g16;
      const bool cv = col < V;  // V is a multiple of 16: a lane's 8 columns are all inside or outside
      const uint32_t co = (uint32_t)col * esz;
      const frag_t<T> af = ld_frag<T>(rs_do, cv ? arow + co : 0x80000000u);
#pragma unroll
      for (int J = 0; J < NB; ++J) {
        if (J <= w) {
          const uint32_t brow = (uint32_t)((16 * J + j16) * V) * esz;
          acc[J] = mma<T>(acc[J], af, ld_frag<T>(rs_v, cv ? brow + co : 0x80000000u));
        }
      }
    }
    // rows 16 w + 4 g16 + r, column 16 J + j16; the causal mask inside the
    // diagonal block, zeros right of it
#pragma unroll
    for (int J = 0; J < NB; ++J)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 4 * g16 + r;
        const float x = (J < w || (J == w && j16 <= row)) ? acc[J][r] : 0.f;
        sdP[(16 * w + row) * LDD + 16 * J + j16] = x;
      }
  }

  // ---- 2. feature groups
  const int lrow = a.sg ? 1 : K;  // gate elements per step
  const T *qc = (const T *)a.q + ((int64_t)bh * T_ + t0) * K;
  const T *kc = (const T *)a.k + ((int64_t)bh * T_ + t0) * K;
  const uint32_t kbytes = rsrc_bytes((int64_t)(T_ - t0) * K * esz);
  const auto rs_q = make_rsrc(qc, kbytes), rs_k = make_rsrc(kc, kbytes);
  // an absent gate (alpha = 1) reads as log alpha = 0 from an empty range
  const auto rs_la = make_rsrc(a.la ? (const T *)a.la + ((int64_t)bh * T_ + t0) * lrow : qc,
                               a.la ? rsrc_bytes((int64_t)(T_ - t0) * lrow * esz) : 0u);
  const auto rs_dqi = make_rsrc((T *)a.dqi + ((int64_t)bh * T_ + t0) * K, kbytes);
  const auto rs_dki = make_rsrc((T *)a.dki + ((int64_t)bh * T_ + t0) * K, kbytes);
  const auto rs_dai = make_rsrc((T *)a.dai + ((int64_t)bh * T_ + t0) * K, kbytes);
  float *datc = a.dat + ((int64_t)bh * a.N + n) * K;
  const int NG = (K + 63) / 64;

  for (int gi = 0; gi < NG; ++gi) {
    const int f = 64 * gi + l;
    const bool fv = f < K;
    // the block's rows of q, k and the gate, for this lane's feature
    uint32_t rq[16], rk[16], rl[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 16 * w + r;
      const uint32_t off = fv ? (uint32_t)((row * K + f) * esz) : 0x80000000u;
      rq[r] = ld_el<T>(rs_q, off);
      rk[r] = ld_el<T>(rs_k, off);
      rl[r] = ld_el<T>(rs_la, a.sg ? (fv ? (uint32_t)(row * esz) : 0x80000000u) : off);
    }
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
    sTot[w * 64 + l] = tot;
    __syncthreads();  // B1: block sums published; the previous group's result tiles are consumed

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
    // for column block J = w, four 16-feature tiles each
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
        const float *ap = sdP + (16 * w + j16) * LDD + 32 * s + 8 * g16;
        const float *bp = sKz + fl * LDD + 32 * s + 8 * g16;
        const f4 a0 = *(const f4 *)ap, a1 = *(const f4 *)(ap + 4);
        const f4 b0 = *(const f4 *)bp, b1 = *(const f4 *)(bp + 4);
        const f8 af = f8{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
        const f8 bf = f8{b0[0] * sc, b0[1] * sc, b0[2] * sc, b0[3] * sc, b1[0] * sc, b1[1] * sc, b1[2] * sc, b1[3] * sc};
        oq[ft] = mma3<T>(oq[ft], af, bf);
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
        f8 af;
#pragma unroll
        for (int u = 0; u < 8; ++u) af[u] = sdP[(32 * s + 8 * g16 + u) * LDD + 16 * w + j16];
        const float *bp = sQz + fl * LDD + 32 * s + 8 * g16;
        const f4 b0 = *(const f4 *)bp, b1 = *(const f4 *)(bp + 4);
        const f8 bf = f8{b0[0] * sc, b0[1] * sc, b0[2] * sc, b0[3] * sc, b1[0] * sc, b1[1] * sc, b1[2] * sc, b1[3] * sc};
        ok[ft] = mma3<T>(ok[ft], af, bf);
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
      st_el<T>(rs_dqi, off, dq);
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

template <typename T, int C, bool PRE>
hipError_t launch_intra_t(const Shape &s, const IntraArgs &a, hipStream_t st) {
  static const hipError_t attr = hipFuncSetAttribute((const void *)intra_kernel<T, C, PRE>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  hipLaunchKernelGGL((intra_kernel<T, C, PRE>), dim3(s.N, s.BH), dim3(64 * (C / 16)), IntraLayout<C>::total, st, a);
  return hipGetLastError();
}

template <typename T, int C>
hipError_t launch_intra_c(const Shape &s, const IntraArgs &a, hipStream_t st) {
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

hipError_t launch_bwd_intra(const Shape &s, const void *q, const void *k, const void *la, const void *v,
                            const void *dO, const Work &w, hipStream_t st) {
  IntraArgs a;
  a.q = q; a.k = k; a.la = la; a.v = v; a.dO = dO;
  a.dqi = w.dqi; a.dki = w.dki; a.dai = w.dai; a.dat = w.dat;
  a.T = s.T; a.K = s.K; a.V = s.V; a.C = s.C; a.N = s.N;
  a.sg = s.sgate ? 1 : 0;
  a.inv_tau = s.inv_tau;
  return s.io == IO_BF16 ? launch_intra_io<bf16>(s, a, st) : launch_intra_io<float>(s, a, st);
}

}  // namespace gla
