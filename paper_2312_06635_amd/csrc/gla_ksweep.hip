// gla_ksweep.hip -- the two backward sweeps that tile the key features (App. B,
// Alg. 4/6 with the corrections listed in the header of gla_vsweep.hip, and the
// closed-form gate gradient of Sec. 4.3).
//
// Per chunk n (S_[n] = state before the chunk, dS_[n+1] = dL/dS after it, B =
// chunk-local inclusive cumsum of log alpha, Lambda = exp(B), Gamma =
// exp(B_last - B), dP = (dO V^T) (.) M):
//   dq_sweep (forward):  dq = Lambda (.) (dO S_[n]^T) + intra(dP, k)
//                        S_[n+1] = Diag(gamma) S_[n] + (K (.) Gamma)^T V
//   dk_sweep (reverse):  dk = Gamma (.) (V dS_[n+1]^T) + intra(dP^T, q)
//                        dS_[n] = Diag(gamma) dS_[n+1] + (Q (.) Lambda)^T dO
//                        dlog alpha = revcumsum(q (.) dq - k (.) dk) + rowsum(S_T (.) dS_T)
// dq, dk and the gate gradient reduce over d_v, so a workgroup owns 32 key
// features of one head for the whole sequence and holds the transposed state
// block (value rows x 32 features, fp32) in matrix-core accumulators.
//
// Workgroup = 8 waves; wave w owns features 16 (w & 1) .. +16 and, in every
// 128-column value slab, value rows 32 (w >> 1) .. +32.  Accumulator pair
// (2 per slab) rows are in the permuted order v = 32 vq + 8 (i / 4) + 4 h +
// i % 4, so the pair is directly an operand whose partner is one contiguous
// 16-byte LDS read.  The products that reduce over d_v leave one partial per
// value quarter; these are pre-scaled, summed in two steps through LDS and
// combined per (row, feature) with the intra-chunk terms:
//   sub-chunk blocks strictly below the diagonal: matrix-core products of fp32
//   operands split into bf16 hi + lo (three cross terms), scaled by the decay
//   of the blocks in between (every exponent <= 0);
//   diagonal blocks: fp32 on the VALUs, factorised exp(B_i - z) exp(z - B_j),
//   or pairwise exp(B_i - B_j) when a block's decay range exceeds kWide.
// Value slabs stream through double-buffered LDS (one barrier per slab).  For
// bf16 the state operand, the gated update operand and the dq hand-off are
// split into bf16 hi + lo so the gate gradient's long reverse sum keeps fp32
// accuracy.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

constexpr int kKT = 512;      // threads per workgroup
constexpr int kKF = 32;       // key features per workgroup
constexpr int kVS = 128;      // value columns per slab
constexpr float kWide = 60.f;

struct KsArgs {
  const void *q, *k, *la, *v, *dO, *dq_in, *dq_lo_in;
  const float *S0, *dST;
  void *dq, *dq_lo, *dk, *dla;
  float *dP, *cST;
  int BH, T, K, V, C, N, KT;
};

template <typename T, int CP> struct KsLayout {
  static constexpr bool DB = sizeof(T) == 2;  // double-buffered slabs (fp32 tiles are too big)
  static constexpr int NBUF = DB ? 2 : 1;
  static constexpr int LDV = kVS;  // slab rows are XOR-swizzled, not padded
  static constexpr int NB = CP / 16, NRG = CP / 4;
  // Per-(row, feature) tiles are stored feature-major ([32 features][rows]),
  // so a factor/final thread's four consecutive rows of one feature and a
  // fragment's eight consecutive rows are single 8/16-byte LDS accesses.
  static constexpr int LDT = CP + 4;                        // fp32 feature-major tiles
  static constexpr int LDTB = CP + (sizeof(T) == 2 ? 8 : 4);  // T feature-major tiles
  static constexpr int LDP = CP + 4;                        // dP (dq: [t][s]; dk: [s][t])
  static constexpr int LDRG = NRG + 4;                      // row-group sums [32][NRG]
  static constexpr size_t slab = sizeof(T) * CP * LDV;
  static constexpr size_t offV = 0;
  static constexpr size_t offD = offV + NBUF * slab;
  static constexpr size_t offBh = offD + NBUF * slab;                    // gated update operand (hi)
  static constexpr size_t offBl = offBh + sizeof(T) * kKF * LDTB;        // (lo, bf16 only)
  static constexpr size_t offO = offBl + (DB ? sizeof(T) * kKF * LDTB : 0);  // orange operand
  static constexpr size_t offPk = offO + 4 * kKF * LDT;                  // pink operand
  static constexpr size_t offBloc = offPk + 4 * kKF * LDT;               // block-local cumsum
  static constexpr size_t offdP = offBloc + 4 * kKF * LDT;
  static constexpr size_t offRed = offdP + 4 * CP * LDP;                 // two partial sums
  static constexpr size_t offOr = offRed + 2 * 4 * kKF * LDT;            // intra-chunk results
  static constexpr size_t offRg = offOr + 4 * kKF * LDT;                 // row-group totals
  static constexpr size_t offSc = offRg + 4 * kKF * LDRG;                // per-block scale [NB][32]
  static constexpr size_t offGp = offSc + 4 * NB * kKF;                  // pair factors [3][32]
  static constexpr size_t offG = offGp + 4 * 3 * kKF;                    // gamma [32]
  static constexpr size_t offCar = offG + 4 * kKF;                       // carry [2][32]
  static constexpr size_t offRedS = offCar + 4 * 2 * kKF;                // final-state sums [8][32]
  static constexpr size_t offFt = offRedS + 4 * 8 * kKF;                 // per-thread block decay [NRG][32]
  static constexpr size_t offGrp = offFt + 4 * NRG * kKF;                // dk: row-group sums of dA
  static constexpr size_t total = offGrp + 4 * kKF * LDRG;
};

// (I, J) of lower-triangular block b (row-major) and of upper block u.
__device__ __forceinline__ void low_block(int b, int &I, int &J) {
  I = (b >= 1) + (b >= 3) + (b >= 6);
  J = b - I * (I + 1) / 2;
}
__device__ __forceinline__ void up_block(int u, int &I, int &J) {
  I = (u >= 3) + (u >= 5);
  J = u - (I == 0 ? -1 : (I == 1 ? 1 : 2));
}
__device__ __forceinline__ int pair_idx(int I, int J) { return I == 2 ? 0 : (J == 0 ? 1 : 2); }

// The permuted-order fragment of ld_col (see gla_vsweep.hip): lane (g, j)
// gets X[r0 + 8g + i][c0 + 8 (j / 4) + 4 h + j % 4].
template <typename T>
__device__ __forceinline__ frag_t<T> ld_col_perm(const T *X, int ld, int r0, int c0, int h) {
  const int l = lane_id(), g = l >> 4, j = l & 15;
  if constexpr (sizeof(T) == 2) {
    const T *p0 = X + (r0 + 8 * g + (j >> 2)) * ld + c0 + 8 * (j & 3) + 4 * h;
    const T *p1 = p0 + 4 * ld;
    s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p0));
    s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p1));
    s8 r = s8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, r);
  } else {
    const T *p = X + (r0 + 8 * g) * ld + c0 + 8 * (j >> 2) + 4 * h + (j & 3);
    f8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = p[i * ld];
    return r;
  }
}

// Slab tiles (V, dO) are stored with their 16-byte chunks XOR-swizzled per
// row, chunk c of row r at c ^ swz(r): both the 16-row fragment reads (one
// chunk of 16 consecutive rows) and the transpose reads (4 rows x 4 chunks)
// then touch distinct LDS banks without padding.
__device__ __forceinline__ int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }
template <typename T> __device__ __forceinline__ int sw_off(int row, int col, int ld) {
  constexpr int EV = 16 / sizeof(T);
  return row * ld + ((col / EV) ^ swz(row)) * EV + col % EV;
}

// ld_row on a swizzled tile: lane (g, j) gets X[r0 + j][c0 + 8g + i].
template <typename T>
__device__ __forceinline__ frag_t<T> ld_row_sw(const T *X, int ld, int r0, int c0) {
  const int l = lane_id(), row = r0 + (l & 15), col = c0 + 8 * (l >> 4);
  if constexpr (sizeof(T) == 2) {
    return *(const bf16x8 *)(X + sw_off<T>(row, col, ld));
  } else {
    const f4 a = *(const f4 *)(X + sw_off<T>(row, col, ld)), b = *(const f4 *)(X + sw_off<T>(row, col + 4, ld));
    return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
}

// ld_col_perm on a swizzled tile.
template <typename T>
__device__ __forceinline__ frag_t<T> ld_col_perm_sw(const T *X, int ld, int r0, int c0, int h) {
  const int l = lane_id(), g = l >> 4, j = l & 15;
  if constexpr (sizeof(T) == 2) {
    const int row = r0 + 8 * g + (j >> 2), col = c0 + 8 * (j & 3) + 4 * h;
    s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(X + sw_off<T>(row, col, ld)));
    s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(X + sw_off<T>(row + 4, col, ld)));
    s8 r = s8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, r);
  } else {
    const int row = r0 + 8 * g, col = c0 + 8 * (j >> 2) + 4 * h + (j & 3);
    f8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = X[sw_off<T>(row + i, col, ld)];
    return r;
  }
}

// Four consecutive elements as one 8-byte (bf16) or 16-byte (fp32) LDS store.
template <typename T> __device__ __forceinline__ void store4(T *p, const T (&v)[4]) {
  if constexpr (sizeof(T) == 2) *(bf16x4 *)p = bf16x4{v[0], v[1], v[2], v[3]};
  else *(f4 *)p = f4{v[0], v[1], v[2], v[3]};
}

// hi + lo = the fp32 accumulator pair to ~16 mantissa bits (lo unused for fp32).
template <typename T>
__device__ __forceinline__ void acc_split(f4 a0, f4 a1, frag_t<T> &hi, frag_t<T> &lo) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi[i] = cvt<T>(a0[i]);
    hi[4 + i] = cvt<T>(a1[i]);
    if constexpr (sizeof(T) == 2) {
      lo[i] = cvt<T>(a0[i] - (float)hi[i]);
      lo[4 + i] = cvt<T>(a1[i] - (float)hi[4 + i]);
    }
  }
}

// fp32 fragment from an fp32 LDS tile: lane (g, j) gets X[r0 + j][c0 + 8g + i].
__device__ __forceinline__ f8 ldf_row(const float *X, int ld, int r0, int c0) {
  const int l = lane_id();
  const float *p = X + (r0 + (l & 15)) * ld + c0 + 8 * (l >> 4);
  const f4 a = *(const f4 *)p, b = *(const f4 *)(p + 4);
  return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// acc += a b for fp32 fragments; on the bf16 path both are split into hi + lo
// and the three significant cross terms are accumulated.
template <typename T> __device__ __forceinline__ f4 mma_split3(f4 acc, const f8 &a, const f8 &b) {
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

template <typename T> __device__ __forceinline__ float elem_f(uint32_t raw) {
  if constexpr (sizeof(T) == 2) return (float)__builtin_bit_cast(bf16, (unsigned short)raw);
  else return __builtin_bit_cast(float, raw);
}
template <typename T> __device__ __forceinline__ uint32_t ld_elem(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
  if constexpr (sizeof(T) == 2) return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
  else return (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
}

// Cumulative-sum bookkeeping of one factor thread (feature fk, rows 4 frg ..
// +3 of the chunk), from the chunk's row-group totals in LDS.
struct Factors {
  float Bloc[4];  // block-local inclusive cumsum of log alpha
  float pre;      // log decay of the blocks before this thread's block
  float tot;      // log decay of this thread's 16-row block
  float blast;    // log decay of the whole chunk
  bool wide;
};

template <int NRG, int LDRG>
__device__ __forceinline__ Factors chunk_factors(const float *sRg, const float (&c)[4], int frg, int fk,
                                                 bool fv) {
  Factors f;
  const int blk = frg >> 2;
  float ex = 0.f;
  f.pre = f.tot = f.blast = 0.f;
  float rg[NRG];
#pragma unroll
  for (int p = 0; p < NRG; p += 4) {
    const f4 v = *(const f4 *)(sRg + fk * LDRG + p);
#pragma unroll
    for (int e = 0; e < 4; ++e) rg[p + e] = v[e];
  }
#pragma unroll
  for (int p = 0; p < NRG; ++p) {
    const float t = rg[p];
    f.blast += t;
    if ((p >> 2) < blk) f.pre += t;
    if ((p >> 2) == blk) {
      f.tot += t;
      if (p < frg) ex += t;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) f.Bloc[i] = ex + c[i];
  f.wide = fv && (-f.tot > kWide);
  return f;
}

// Per-chunk gate data every factor thread publishes: exp of the block-level
// scale, gamma and the decays between non-adjacent blocks.
template <int NB, int LDRG>
__device__ __forceinline__ void publish_decays(float *sSc, float *sG, float *sGp, const float *sRg,
                                               const Factors &f, float scale_log, int frg, int fk,
                                               bool fv) {
  if ((frg & 3) == 0) sSc[(frg >> 2) * kKF + fk] = __expf(scale_log);
  if (frg == 0) {
    sG[fk] = fv ? __expf(f.blast) : 0.f;
    if constexpr (NB == 4) {
      float t1 = 0.f, t2 = 0.f;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        t1 += sRg[fk * LDRG + 4 + p];
        t2 += sRg[fk * LDRG + 8 + p];
      }
      sGp[0 * kKF + fk] = __expf(t1);
      sGp[1 * kKF + fk] = __expf(t1 + t2);
      sGp[2 * kKF + fk] = __expf(t2);
    }
  }
}

// ============================================================== dq sweep
template <typename T, int CP, int NSL>
__global__ void __launch_bounds__(kKT) dq_sweep_kernel(KsArgs a) {
  using L = KsLayout<T, CP>;
  constexpr int NB = L::NB, NRG = L::NRG, NSC = CP / 32, NBLK = NB * (NB + 1) / 2;
  constexpr int NUP = NB * (NB - 1) / 2;
  constexpr bool SPLIT = sizeof(T) == 2;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T *sV0 = (T *)(smem + L::offV), *sD0 = (T *)(smem + L::offD);
  T *sBh = (T *)(smem + L::offBh), *sBl = (T *)(smem + L::offBl);
  float *sKo = (float *)(smem + L::offO), *sKp = (float *)(smem + L::offPk);
  float *sBloc = (float *)(smem + L::offBloc), *sdP = (float *)(smem + L::offdP);
  float *sRed = (float *)(smem + L::offRed), *sOr = (float *)(smem + L::offOr);
  float *sRg = (float *)(smem + L::offRg), *sSc = (float *)(smem + L::offSc);
  float *sGp = (float *)(smem + L::offGp), *sG = (float *)(smem + L::offG);
  float *sRedS = (float *)(smem + L::offRedS), *sFt = (float *)(smem + L::offFt);

  int bh, kt;
  xcd_map(a.BH, a.KT, bh, kt);
  const int tid = threadIdx.x, w = wave_id(), l = lane_id(), g = l >> 4, j = l & 15;
  const int kb = w & 1, vq = w >> 1;
  const int K = a.K, V = a.V, C = a.C, N = a.N, k0 = kt * kKF;
  const int fk = tid & 31, frg = tid >> 5;
  const bool fthr = frg < NRG;
  const int kf = k0 + fk;
  const bool fv = kf < K;
  const int esz = sizeof(T);

  for (int i = tid; i < CP * L::LDP; i += kKT) sdP[i] = 0.f;

  f4 S[NSL][2];
#pragma unroll
  for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int vv = sl * kVS + 32 * vq + 8 * g + 4 * h + r, kq = k0 + 16 * kb + j;
        S[sl][h][r] = (a.S0 && vv < V && kq < K) ? a.S0[((int64_t)bh * K + kq) * V + vv] : 0.f;
      }

  // ---- input streams
  const T *kh_ = (const T *)a.k + (int64_t)bh * a.T * K, *lah = (const T *)a.la + (int64_t)bh * a.T * K;
  const T *vh = (const T *)a.v + (int64_t)bh * a.T * V, *dOh = (const T *)a.dO + (int64_t)bh * a.T * V;
  uint32_t eoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * frg + i;
    eoff[i] = (fthr && row < C && fv) ? (uint32_t)((row * K + kf) * esz) : 0x80000000u;
  }
  uint32_t fin_la[4], fin_k[4];
  auto fetch_factors = [&](int n) {
    const int t0 = n * C;
    const auto rs_la = make_rsrc(lah + (int64_t)t0 * K, rsrc_bytes((int64_t)(a.T - t0) * K * esz));
    const auto rs_k = make_rsrc(kh_ + (int64_t)t0 * K, rsrc_bytes((int64_t)(a.T - t0) * K * esz));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fin_la[i] = ld_elem<T>(rs_la, eoff[i]);
      fin_k[i] = ld_elem<T>(rs_k, eoff[i]);
    }
  };
  TileLd<T, CP, kVS, kKT> pv, pd;
  pv.init(V, C, kVS);
  pd.init(V, C, kVS);
  const int NQ = N * NSL;
  auto fetch_slab = [&](int q) {
    if (q >= NQ) return;
    const int n = q / NSL, sl = q - n * NSL, t0 = n * C, c0 = sl * kVS;
    const uint32_t bytes = rsrc_bytes(((int64_t)(a.T - t0) * V - c0) * esz);
    pv.load(make_rsrc(vh + (int64_t)t0 * V + c0, bytes), V - c0);
    pd.load(make_rsrc(dOh + (int64_t)t0 * V + c0, bytes), V - c0);
  };
  auto store_slab = [&](int q) {
    const int b = L::DB ? (q & 1) : 0;
    pv.store_swz((T *)((char *)sV0 + b * L::slab), L::LDV);
    pd.store_swz((T *)((char *)sD0 + b * L::slab), L::LDV);
  };

  T *dqo = (T *)a.dq + (int64_t)bh * a.T * K, *dqlo = (T *)a.dq_lo + (int64_t)bh * a.T * K;
  float *dPg = a.dP + (int64_t)bh * N * C * C;

  fetch_factors(0);
  fetch_slab(0);
  if constexpr (L::DB) {
    store_slab(0);
    fetch_slab(1);
  }

  for (int n = 0; n < N; ++n) {
    const int t0 = n * C, rv = min(C, a.T - t0);
    // ---- factors: cumsum of log alpha, gated operands
    float c[4], kv[4];
    {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s += elem_f<T>(fin_la[i]);
        c[i] = s;
        kv[i] = elem_f<T>(fin_k[i]);
      }
      if (fthr) sRg[fk * L::LDRG + frg] = s;
    }
    __syncthreads();
    if (fthr) {
      const Factors f = chunk_factors<NRG, L::LDRG>(sRg, c, frg, fk, fv);
      sFt[frg * kKF + fk] = f.tot;
      const float etot = __expf(-f.tot), ekt = __expf(f.blast - f.pre - f.tot);
      f4 ko4, kp4, bl4;
      T hi4[4], lo4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float ks = kv[i] * __expf(f.tot - f.Bloc[i]);
        const float kt_ = ks * ekt;
        hi4[i] = cvt<T>(kt_);
        lo4[i] = cvt<T>(kt_ - (float)hi4[i]);
        ko4[i] = ks;
        kp4[i] = f.wide ? 0.f : ks * etot;
        bl4[i] = f.Bloc[i];
      }
      store4<T>(sBh + fk * L::LDTB + 4 * frg, hi4);
      if constexpr (SPLIT) store4<T>(sBl + fk * L::LDTB + 4 * frg, lo4);
      *(f4 *)(sKo + fk * L::LDT + 4 * frg) = ko4;
      *(f4 *)(sKp + fk * L::LDT + 4 * frg) = kp4;
      *(f4 *)(sBloc + fk * L::LDT + 4 * frg) = bl4;
      publish_decays<NB, L::LDRG>(sSc, sG, sGp, sRg, f, f.pre, frg, fk, fv);
    }
    if (n + 1 < N) fetch_factors(n + 1);
    __syncthreads();

    // ---- slabs: dP blocks, dq_inter partials (state before the chunk), update
    frag_t<T> bh_[NSC], bl_[NSC];
#pragma unroll
    for (int sc = 0; sc < NSC; ++sc) {
      bh_[sc] = ld_row<T>(sBh, L::LDTB, 16 * kb, 32 * sc);
      if constexpr (SPLIT) bl_[sc] = ld_row<T>(sBl, L::LDTB, 16 * kb, 32 * sc);
    }
    const float gam = sG[16 * kb + j];
    f4 acc[NB], accP[2];
#pragma unroll
    for (int I = 0; I < NB; ++I) acc[I] = zero4();
    accP[0] = accP[1] = zero4();
    int pI0, pJ0, pI1, pJ1;
    low_block(w, pI0, pJ0);
    low_block(w + 8, pI1, pJ1);
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl) {
      const int q = n * NSL + sl;
      if constexpr (!L::DB) {
        store_slab(q);
        fetch_slab(q + 1);
        __syncthreads();
      }
      const int b = L::DB ? (q & 1) : 0;
      const T *sV = (const T *)((const char *)sV0 + b * L::slab);
      const T *sD = (const T *)((const char *)sD0 + b * L::slab);
      if (sl * kVS < V) {
        // dP = dO V^T over this slab, for this wave's blocks
        if (w < NBLK) {
#pragma unroll
          for (int s = 0; s < kVS / 32; ++s)
            accP[0] = mma<T>(accP[0], ld_row_sw<T>(sD, L::LDV, 16 * pI0, 32 * s), ld_row_sw<T>(sV, L::LDV, 16 * pJ0, 32 * s));
        }
        if (w + 8 < NBLK) {
#pragma unroll
          for (int s = 0; s < kVS / 32; ++s)
            accP[1] = mma<T>(accP[1], ld_row_sw<T>(sD, L::LDV, 16 * pI1, 32 * s), ld_row_sw<T>(sV, L::LDV, 16 * pJ1, 32 * s));
        }
        // dq_inter += dO[:, this wave's 32 value rows] S^T
        frag_t<T> shi, slo;
        acc_split<T>(S[sl][0], S[sl][1], shi, slo);
#pragma unroll
        for (int I = 0; I < NB; ++I) {
          const frag_t<T> ad = ld_row_sw<T>(sD, L::LDV, 16 * I, 32 * vq);
          acc[I] = mma<T>(acc[I], ad, shi);
          if constexpr (SPLIT) acc[I] = mma<T>(acc[I], ad, slo);
        }
        // S^T <- gamma S^T + V^T (K (.) Gamma)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          S[sl][h] *= gam;
#pragma unroll
          for (int sc = 0; sc < NSC; ++sc) {
            const frag_t<T> av = ld_col_perm_sw<T>(sV, L::LDV, 32 * sc, 32 * vq, h);
            S[sl][h] = mma<T>(S[sl][h], av, bh_[sc]);
            if constexpr (SPLIT) S[sl][h] = mma<T>(S[sl][h], av, bl_[sc]);
          }
        }
      }
      if constexpr (L::DB) {
        store_slab(q + 1);
        fetch_slab(q + 2);
      }
      __syncthreads();
    }

    // ---- dP to LDS (and to the workspace for the dk sweep)
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int bI = u ? pI1 : pI0, bJ = u ? pJ1 : pJ0;
      if (w + 8 * u < NBLK) {
        const int t4 = 16 * bI + 4 * g, col = 16 * bJ + j;
        f4 v4;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v4[r] = col > t4 + r ? 0.f : accP[u][r];
          sdP[(t4 + r) * L::LDP + col] = v4[r];
        }
        // the workspace holds dP transposed ([s][t]) for the dk sweep
        if (kt == 0 && t4 < C && col < C) *(f4 *)(dPg + ((int64_t)n * C + col) * C + t4) = v4;
      }
    }
    if (kt == 0 && w < NUP) {
      int uI, uJ;
      up_block(w, uI, uJ);
      const int t4 = 16 * uI + 4 * g, col = 16 * uJ + j;
      if (t4 < C && col < C) *(f4 *)(dPg + ((int64_t)n * C + col) * C + t4) = zero4();
    }
    // ---- dq_inter partials, pre-scaled by exp(log decay before the block)
#pragma unroll
    for (int I = 0; I < NB; ++I) acc[I] *= sSc[I * kKF + 16 * kb + j];
    if (vq >= 2) {
#pragma unroll
      for (int I = 0; I < NB; ++I) *(f4 *)(sRed + ((vq - 2) * kKF + 16 * kb + j) * L::LDT + 16 * I + 4 * g) = acc[I];
    }
    __syncthreads();
    if (vq < 2) {
#pragma unroll
      for (int I = 0; I < NB; ++I) *(f4 *)(sRed + (vq * kKF + 16 * kb + j) * L::LDT + 16 * I + 4 * g) += acc[I];
    }
    // intra-chunk term by sub-chunk blocks, for row block I: sum over J <= I of
    // dP_IJ x_J with x_J = (k (.) exp(tot_J - Bloc)) g_IJ below the diagonal and
    // k (.) exp(-Bloc) on it (zero where the block needs pairwise decays)
    for (int t = w; t < 2 * NB; t += 8) {
      const int I = t >> 1, kq = t & 1;
      f4 o = zero4();
#pragma unroll
      for (int s = 0; s < NSC; ++s) {
        if (32 * s > 16 * I) continue;
        const int J = 2 * s + (g >> 1);
        const float sc = J > I ? 0.f : (J <= I - 2 ? sGp[pair_idx(I, J) * kKF + 16 * kq + j] : 1.f);
        const f8 ko = ldf_row(sKo, L::LDT, 16 * kq, 32 * s), kp = ldf_row(sKp, L::LDT, 16 * kq, 32 * s);
        f8 bf;
#pragma unroll
        for (int i = 0; i < 8; ++i) bf[i] = J == I ? kp[i] : ko[i] * sc;
        o = mma_split3<T>(o, ldf_row(sdP, L::LDP, 16 * I, 32 * s), bf);
      }
      *(f4 *)(sOr + (16 * kq + j) * L::LDT + 16 * I + 4 * g) = o;
    }
    __syncthreads();

    // ---- dq = Lambda (.) inter + intra, per (row, feature)
    if (fthr) {
      const int blk = frg >> 2;
      const bool wide = fv && (-sFt[frg * kKF + fk] > kWide);
      const f4 r0 = *(const f4 *)(sRed + fk * L::LDT + 4 * frg);
      const f4 r1 = *(const f4 *)(sRed + (kKF + fk) * L::LDT + 4 * frg);
      const f4 op = *(const f4 *)(sOr + fk * L::LDT + 4 * frg);
      const f4 bl4 = *(const f4 *)(sBloc + fk * L::LDT + 4 * frg);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * frg + i;
        const float bloc = bl4[i];
        float dq = __expf(bloc) * (r0[i] + r1[i] + op[i]);
        if (wide && row < rv) {
          // diagonal block with pairwise decays exp(B_row - B_s)
#pragma unroll 1
          for (int s = 16 * blk; s <= row; ++s)
            dq += sdP[row * L::LDP + s] * (float)kh_[(int64_t)(t0 + s) * K + kf] *
                  __expf(bloc - sBloc[fk * L::LDT + s]);
        }
        if (row < rv && fv) {
          const T hi = cvt<T>(dq);
          dqo[(int64_t)(t0 + row) * K + kf] = hi;
          if constexpr (SPLIT) dqlo[(int64_t)(t0 + row) * K + kf] = cvt<T>(dq - (float)hi);
        }
      }
    }
  }

  // ---- final-state term of the gate gradient: rowsum(S_T (.) dS_T) per feature
  if (a.dST) {
    float part = 0.f;
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int vv = sl * kVS + 32 * vq + 8 * g + 4 * h + r, kq = k0 + 16 * kb + j;
          if (vv < V && kq < K) part += S[sl][h][r] * a.dST[((int64_t)bh * K + kq) * V + vv];
        }
    part += __shfl_xor(part, 16);
    part += __shfl_xor(part, 32);
    if (g == 0) sRedS[w * kKF + j] = part;
    __syncthreads();
    if (tid < kKF && k0 + tid < K) {
      const int kq = tid >> 4, jj = tid & 15;
      float s = 0.f;
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) s += sRedS[(2 * v4 + kq) * kKF + jj];
      a.cST[(int64_t)bh * K + k0 + tid] = s;
    }
  }
}

// ============================================================== dk sweep
template <typename T, int CP, int NSL>
__global__ void __launch_bounds__(kKT) dk_sweep_kernel(KsArgs a) {
  using L = KsLayout<T, CP>;
  constexpr int NB = L::NB, NRG = L::NRG, NSC = CP / 32;
  constexpr bool SPLIT = sizeof(T) == 2;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T *sV0 = (T *)(smem + L::offV), *sD0 = (T *)(smem + L::offD);
  T *sBh = (T *)(smem + L::offBh), *sBl = (T *)(smem + L::offBl);
  float *sQo = (float *)(smem + L::offO), *sQp = (float *)(smem + L::offPk);
  float *sBloc = (float *)(smem + L::offBloc), *sdP = (float *)(smem + L::offdP);
  float *sRed = (float *)(smem + L::offRed), *sOr = (float *)(smem + L::offOr);
  float *sRg = (float *)(smem + L::offRg), *sSc = (float *)(smem + L::offSc);
  float *sGp = (float *)(smem + L::offGp), *sG = (float *)(smem + L::offG);
  float *sCar = (float *)(smem + L::offCar), *sFt = (float *)(smem + L::offFt);
  float *sGrp = (float *)(smem + L::offGrp);

  int bh, kt;
  xcd_map(a.BH, a.KT, bh, kt);
  const int tid = threadIdx.x, w = wave_id(), l = lane_id(), g = l >> 4, j = l & 15;
  const int kb = w & 1, vq = w >> 1;
  const int K = a.K, V = a.V, C = a.C, N = a.N, k0 = kt * kKF;
  const int fk = tid & 31, frg = tid >> 5;
  const bool fthr = frg < NRG;
  const int kf = k0 + fk;
  const bool fv = kf < K;
  const int esz = sizeof(T);

  if (tid < kKF) sCar[tid] = (a.cST && k0 + tid < K) ? a.cST[(int64_t)bh * K + k0 + tid] : 0.f;

  f4 dS[NSL][2];
#pragma unroll
  for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int vv = sl * kVS + 32 * vq + 8 * g + 4 * h + r, kq = k0 + 16 * kb + j;
        dS[sl][h][r] = (a.dST && vv < V && kq < K) ? a.dST[((int64_t)bh * K + kq) * V + vv] : 0.f;
      }

  const T *qh_ = (const T *)a.q + (int64_t)bh * a.T * K, *kh_ = (const T *)a.k + (int64_t)bh * a.T * K;
  const T *lah = (const T *)a.la + (int64_t)bh * a.T * K;
  const T *dqh = (const T *)a.dq_in + (int64_t)bh * a.T * K;
  const T *dqlh = SPLIT ? (const T *)a.dq_lo_in + (int64_t)bh * a.T * K : dqh;
  const T *vh = (const T *)a.v + (int64_t)bh * a.T * V, *dOh = (const T *)a.dO + (int64_t)bh * a.T * V;
  const float *dPg = a.dP + (int64_t)bh * N * C * C;
  uint32_t eoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * frg + i;
    eoff[i] = (fthr && row < C && fv) ? (uint32_t)((row * K + kf) * esz) : 0x80000000u;
  }
  uint32_t fin_la[4], fin_q[4], fin_k[4], fin_dq[4], fin_dql[4];
  TileLd<float, CP, CP, kKT> pp;
  pp.init(C, C, C);
  auto fetch_factors = [&](int n) {
    const int t0 = n * C;
    const uint32_t bytes = rsrc_bytes((int64_t)(a.T - t0) * K * esz);
    const auto rs_la = make_rsrc(lah + (int64_t)t0 * K, bytes);
    const auto rs_q = make_rsrc(qh_ + (int64_t)t0 * K, bytes);
    const auto rs_k = make_rsrc(kh_ + (int64_t)t0 * K, bytes);
    const auto rs_dq = make_rsrc(dqh + (int64_t)t0 * K, bytes);
    const auto rs_dql = make_rsrc(dqlh + (int64_t)t0 * K, bytes);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fin_la[i] = ld_elem<T>(rs_la, eoff[i]);
      fin_q[i] = ld_elem<T>(rs_q, eoff[i]);
      fin_k[i] = ld_elem<T>(rs_k, eoff[i]);
      fin_dq[i] = ld_elem<T>(rs_dq, eoff[i]);
      fin_dql[i] = SPLIT ? ld_elem<T>(rs_dql, eoff[i]) : 0u;
    }
    pp.load(make_rsrc(dPg + (int64_t)n * C * C, (uint32_t)(C * C * 4)));
  };
  TileLd<T, CP, kVS, kKT> pv, pd;
  pv.init(V, C, kVS);
  pd.init(V, C, kVS);
  const int NQ = N * NSL;
  auto fetch_slab = [&](int q) {
    if (q >= NQ) return;
    const int n = N - 1 - q / NSL, sl = q % NSL, t0 = n * C, c0 = sl * kVS;
    const uint32_t bytes = rsrc_bytes(((int64_t)(a.T - t0) * V - c0) * esz);
    pv.load(make_rsrc(vh + (int64_t)t0 * V + c0, bytes), V - c0);
    pd.load(make_rsrc(dOh + (int64_t)t0 * V + c0, bytes), V - c0);
  };
  auto store_slab = [&](int q) {
    const int b = L::DB ? (q & 1) : 0;
    pv.store_swz((T *)((char *)sV0 + b * L::slab), L::LDV);
    pd.store_swz((T *)((char *)sD0 + b * L::slab), L::LDV);
  };

  T *dko = (T *)a.dk + (int64_t)bh * a.T * K, *dlao = (T *)a.dla + (int64_t)bh * a.T * K;

  fetch_factors(N - 1);
  fetch_slab(0);
  if constexpr (L::DB) {
    store_slab(0);
    fetch_slab(1);
  }

  for (int it = 0; it < N; ++it) {
    const int n = N - 1 - it;
    const int t0 = n * C, rv = min(C, a.T - t0);
    // ---- factors
    float c[4], qv[4], kv[4], qdq[4];
    {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s += elem_f<T>(fin_la[i]);
        c[i] = s;
        qv[i] = elem_f<T>(fin_q[i]);
        kv[i] = elem_f<T>(fin_k[i]);
        qdq[i] = qv[i] * (elem_f<T>(fin_dq[i]) + (SPLIT ? elem_f<T>(fin_dql[i]) : 0.f));
      }
      if (fthr) sRg[fk * L::LDRG + frg] = s;
      pp.store(sdP, L::LDP);
    }
    __syncthreads();
    if (fthr) {
      const Factors f = chunk_factors<NRG, L::LDRG>(sRg, c, frg, fk, fv);
      sFt[frg * kKF + fk] = f.tot;
      const float epre = __expf(f.pre), etot = __expf(-f.tot);
      f4 qo4, qp4, bl4;
      T hi4[4], lo4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float qh = qv[i] * __expf(f.Bloc[i]);
        const float qt = qh * epre;
        hi4[i] = cvt<T>(qt);
        lo4[i] = cvt<T>(qt - (float)hi4[i]);
        qo4[i] = qh;
        qp4[i] = f.wide ? 0.f : qh * etot;
        bl4[i] = f.Bloc[i];
      }
      store4<T>(sBh + fk * L::LDTB + 4 * frg, hi4);
      if constexpr (SPLIT) store4<T>(sBl + fk * L::LDTB + 4 * frg, lo4);
      *(f4 *)(sQo + fk * L::LDT + 4 * frg) = qo4;
      *(f4 *)(sQp + fk * L::LDT + 4 * frg) = qp4;
      *(f4 *)(sBloc + fk * L::LDT + 4 * frg) = bl4;
      publish_decays<NB, L::LDRG>(sSc, sG, sGp, sRg, f, f.blast - f.pre - f.tot, frg, fk, fv);
    }
    if (it + 1 < N) fetch_factors(n - 1);
    __syncthreads();

    // ---- slabs: dk_inter partials (dS after the chunk), then the dS update
    frag_t<T> bh_[NSC], bl_[NSC];
#pragma unroll
    for (int sc = 0; sc < NSC; ++sc) {
      bh_[sc] = ld_row<T>(sBh, L::LDTB, 16 * kb, 32 * sc);
      if constexpr (SPLIT) bl_[sc] = ld_row<T>(sBl, L::LDTB, 16 * kb, 32 * sc);
    }
    const float gam = sG[16 * kb + j];
    f4 acc[NB];
#pragma unroll
    for (int J = 0; J < NB; ++J) acc[J] = zero4();
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl) {
      const int q = it * NSL + sl;
      if constexpr (!L::DB) {
        store_slab(q);
        fetch_slab(q + 1);
        __syncthreads();
      }
      const int b = L::DB ? (q & 1) : 0;
      const T *sV = (const T *)((const char *)sV0 + b * L::slab);
      const T *sD = (const T *)((const char *)sD0 + b * L::slab);
      if (sl * kVS < V) {
        frag_t<T> shi, slo;
        acc_split<T>(dS[sl][0], dS[sl][1], shi, slo);
#pragma unroll
        for (int J = 0; J < NB; ++J) {
          const frag_t<T> av = ld_row_sw<T>(sV, L::LDV, 16 * J, 32 * vq);
          acc[J] = mma<T>(acc[J], av, shi);
          if constexpr (SPLIT) acc[J] = mma<T>(acc[J], av, slo);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          dS[sl][h] *= gam;
#pragma unroll
          for (int sc = 0; sc < NSC; ++sc) {
            const frag_t<T> ad = ld_col_perm_sw<T>(sD, L::LDV, 32 * sc, 32 * vq, h);
            dS[sl][h] = mma<T>(dS[sl][h], ad, bh_[sc]);
            if constexpr (SPLIT) dS[sl][h] = mma<T>(dS[sl][h], ad, bl_[sc]);
          }
        }
      }
      if constexpr (L::DB) {
        store_slab(q + 1);
        fetch_slab(q + 2);
      }
      __syncthreads();
    }

    // ---- dk_inter partials, pre-scaled by exp(B_last - B at the block's end)
#pragma unroll
    for (int J = 0; J < NB; ++J) acc[J] *= sSc[J * kKF + 16 * kb + j];
    if (vq >= 2) {
#pragma unroll
      for (int J = 0; J < NB; ++J) *(f4 *)(sRed + ((vq - 2) * kKF + 16 * kb + j) * L::LDT + 16 * J + 4 * g) = acc[J];
    }
    __syncthreads();
    if (vq < 2) {
#pragma unroll
      for (int J = 0; J < NB; ++J) *(f4 *)(sRed + (vq * kKF + 16 * kb + j) * L::LDT + 16 * J + 4 * g) += acc[J];
    }
    // intra-chunk term by sub-chunk blocks, for column block J: sum over I >= J
    // of dP_IJ^T y_I with y_I = (q (.) exp(Bloc)) g_IJ below the diagonal and
    // q (.) exp(Bloc - tot_J) on it (zero where the block needs pairwise decays)
    for (int t = w; t < 2 * NB; t += 8) {
      const int J = t >> 1, kq = t & 1;
      f4 o = zero4();
#pragma unroll
      for (int s = 0; s < NSC; ++s) {
        if (32 * s + 31 < 16 * J) continue;
        const int I = 2 * s + (g >> 1);
        const float sc = I < J ? 0.f : (I >= J + 2 ? sGp[pair_idx(I, J) * kKF + 16 * kq + j] : 1.f);
        const f8 qo = ldf_row(sQo, L::LDT, 16 * kq, 32 * s), qp = ldf_row(sQp, L::LDT, 16 * kq, 32 * s);
        f8 bf;
#pragma unroll
        for (int i = 0; i < 8; ++i) bf[i] = I == J ? qp[i] : qo[i] * sc;
        o = mma_split3<T>(o, ldf_row(sdP, L::LDP, 16 * J, 32 * s), bf);
      }
      *(f4 *)(sOr + (16 * kq + j) * L::LDT + 16 * J + 4 * g) = o;
    }
    __syncthreads();

    // ---- dk = Gamma (.) inter + intra; dA = q dq - k dk; in-chunk reverse sums
    float dA[4];
    if (fthr) {
      const int blk = frg >> 2;
      const float tot = sFt[frg * kKF + fk];
      const bool wide = fv && (-tot > kWide);
      const f4 r0 = *(const f4 *)(sRed + fk * L::LDT + 4 * frg);
      const f4 r1 = *(const f4 *)(sRed + (kKF + fk) * L::LDT + 4 * frg);
      const f4 op = *(const f4 *)(sOr + fk * L::LDT + 4 * frg);
      const f4 bl4 = *(const f4 *)(sBloc + fk * L::LDT + 4 * frg);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * frg + i;
        const float bloc = bl4[i];
        float dk = __expf(tot - bloc) * (r0[i] + r1[i] + op[i]);
        if (wide && row < rv) {
          // diagonal block with pairwise decays exp(B_t - B_row)
          const int tend = min(16 * blk + 16, rv);
#pragma unroll 1
          for (int tt = row; tt < tend; ++tt)
            dk += sdP[row * L::LDP + tt] * (float)qh_[(int64_t)(t0 + tt) * K + kf] *
                  __expf(sBloc[fk * L::LDT + tt] - bloc);
        }
        dA[i] = qdq[i] - kv[i] * dk;
        if (row < rv && fv) dko[(int64_t)(t0 + row) * K + kf] = cvt<T>(dk);
      }
      float s = 0.f;
#pragma unroll
      for (int i = 3; i >= 0; --i) {
        s += dA[i];
        dA[i] = s;
      }
      sGrp[fk * L::LDRG + frg] = s;
    }
    __syncthreads();
    if (fthr) {
      const float *car = sCar + (it & 1) * kKF;
      float later = car[fk], all = car[fk];
#pragma unroll
      for (int p = 0; p < NRG; p += 4) {
        const f4 v = *(const f4 *)(sGrp + fk * L::LDRG + p);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          all += v[e];
          if (p + e > frg) later += v[e];
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 4 * frg + i;
        if (row < rv && fv) dlao[(int64_t)(t0 + row) * K + kf] = cvt<T>(dA[i] + later);
      }
      if (frg == 0) sCar[((it + 1) & 1) * kKF + fk] = all;
    }
    __syncthreads();
  }
}

// ============================================================== launchers
int ks_cp(const Shape &s) { return s.C <= 32 ? 32 : 64; }
int ks_nsl(const Shape &s) {
  const int n = (s.V + kVS - 1) / kVS;
  return n <= 1 ? 1 : (n <= 2 ? 2 : (n <= 4 ? 4 : 8));
}

template <typename T, int CP> size_t ks_lds_t() { return KsLayout<T, CP>::total; }

size_t ks_lds(const Shape &s) {
  const bool b = s.io == IO_BF16;
  if (ks_cp(s) == 32) return b ? ks_lds_t<bf16, 32>() : ks_lds_t<float, 32>();
  return b ? ks_lds_t<bf16, 64>() : ks_lds_t<float, 64>();
}

KsArgs ks_args(const Shape &s) {
  KsArgs a{};
  a.BH = s.BH; a.T = s.T; a.K = s.K; a.V = s.V; a.C = s.C; a.N = s.N;
  a.KT = (s.K + kKF - 1) / kKF;
  return a;
}

template <bool DQ, typename T, int CP, int NSL>
hipError_t launch_ks_t(const KsArgs &a, hipStream_t st) {
  static bool attr = false;
  const size_t lds = KsLayout<T, CP>::total;
  const void *fn = DQ ? (const void *)dq_sweep_kernel<T, CP, NSL> : (const void *)dk_sweep_kernel<T, CP, NSL>;
  if (!attr) {
    (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr = true;
  }
  if constexpr (DQ)
    hipLaunchKernelGGL((dq_sweep_kernel<T, CP, NSL>), dim3(a.BH * a.KT), dim3(kKT), lds, st, a);
  else
    hipLaunchKernelGGL((dk_sweep_kernel<T, CP, NSL>), dim3(a.BH * a.KT), dim3(kKT), lds, st, a);
  return hipGetLastError();
}

template <bool DQ, typename T, int CP>
hipError_t dispatch_ks_cp(const Shape &s, const KsArgs &a, hipStream_t st) {
  switch (ks_nsl(s)) {
    case 1: return launch_ks_t<DQ, T, CP, 1>(a, st);
    case 2: return launch_ks_t<DQ, T, CP, 2>(a, st);
    case 4: return launch_ks_t<DQ, T, CP, 4>(a, st);
    default: return launch_ks_t<DQ, T, CP, 8>(a, st);
  }
}

template <bool DQ>
hipError_t dispatch_ks(const Shape &s, const KsArgs &a, hipStream_t st) {
  if (s.io == IO_BF16)
    return ks_cp(s) == 32 ? dispatch_ks_cp<DQ, bf16, 32>(s, a, st) : dispatch_ks_cp<DQ, bf16, 64>(s, a, st);
  return ks_cp(s) == 32 ? dispatch_ks_cp<DQ, float, 32>(s, a, st) : dispatch_ks_cp<DQ, float, 64>(s, a, st);
}

}  // namespace

size_t lds_bwd_dq(const Shape &s) { return ks_lds(s); }
size_t lds_bwd_dk(const Shape &s) { return ks_lds(s); }

hipError_t launch_bwd_dq(const Shape &s, const void *k, const void *la, const void *v,
                         const float *S0, const void *dO, const float *dST, void *dq,
                         const Work &w, hipStream_t st) {
  KsArgs a = ks_args(s);
  a.k = k; a.la = la; a.v = v; a.dO = dO; a.S0 = S0; a.dST = dST; a.dq = dq; a.dq_lo = w.dq_lo;
  a.dP = w.dP; a.cST = w.cST;
  if (s.io != IO_BF16) a.dq_lo = dq;  // unused
  return dispatch_ks<true>(s, a, st);
}

hipError_t launch_bwd_dk(const Shape &s, const void *q, const void *k, const void *la,
                         const void *v, const void *dO, const float *dST, const void *dq,
                         void *dk, void *dla, const Work &w, hipStream_t st) {
  KsArgs a = ks_args(s);
  a.q = q; a.k = k; a.la = la; a.v = v; a.dO = dO; a.dST = dST; a.dq_in = dq; a.dq_lo_in = w.dq_lo;
  a.dk = dk; a.dla = dla; a.dP = w.dP; a.cST = dST ? w.cST : nullptr;
  return dispatch_ks<false>(s, a, st);
}

}  // namespace gla
