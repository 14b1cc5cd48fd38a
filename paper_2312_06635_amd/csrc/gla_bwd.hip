// gla_bwd.hip -- backward of the chunkwise GLA form (App. B, Alg. 4/6 with the
// typos corrected, and the closed-form gate gradient of Sec. 4.3).
//
// Per chunk n (states S_[n] before the chunk, dS_[n+1] = dL/dS after it):
//   dq = Lambda (.) (dO S_[n]^T)        + intra(dP, k)
//   dk = Gamma  (.) (V dS_[n+1]^T)      + intra(dP^T, q)
//   dv = (K (.) Gamma) dS_[n+1]         + P^T dO
//   dS_[n] = Diag(gamma) dS_[n+1] + (Q (.) Lambda)^T dO,   dP = (dO V^T) (.) M
//   dlog alpha = revcumsum(q (.) dq - k (.) dk) + rowsum(S_T (.) dS_T)
// The gate scales the rows (key features) of the state, so dq, dk and the
// gate gradient are local to a block of key features ("K-tiled", reduction
// over d_v inside the workgroup), while dv is local to a block of value
// columns ("V-tiled").  Three sweeps:
//   bwd_dq : K-tiled, forward in time; recomputes S (Sec. 3.3) and writes dq
//            (and dP, which it needs anyway, for bwd_dk)
//   bwd_dk : K-tiled, backward in time; dS, dk and dlog alpha (the reverse
//            cumulative sum is carried across chunks)
//   bwd_dv : V-tiled, backward in time; dS and dv
// In the K-tiled sweeps the state block is kept transposed (rows = value
// columns, cols = 32 key features) so that products reducing over d_v can take
// it directly as a matrix-core operand.  Intra-chunk terms use the same
// block-boundary normalisation as the forward: 16x16 blocks strictly below
// the diagonal on the matrix cores, diagonal blocks in fp32 on the VALUs.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

constexpr float kWideRangeB = 60.0f;

static int round_up(int x, int m) { return (x + m - 1) / m * m; }
// Smallest power of two >= max(x, lo) (tile widths must be powers of two).
static int pow2_at_least(int x, int lo) {
  int p = lo;
  while (p < x) p *= 2;
  return p;
}

__device__ __forceinline__ int pair_idx(int I, int J) { return I == 2 ? 0 : (J == 0 ? 1 : 2); }

// (I, J) of the b-th lower-triangular 16x16 block, row-major.
__device__ __forceinline__ void tri_block(int b, int &I, int &J) {
  I = 0;
  while ((I + 1) * (I + 2) / 2 <= b) ++I;
  J = b - I * (I + 1) / 2;
}

struct KArgs {
  const void *q, *k, *la, *v, *dO, *dq_in, *dq_lo_in;
  const float *S0, *dST;
  void *dq, *dq_lo, *dk, *dla;
  float *dP, *cST;
  int BH, T, K, V, C, Cp, N, KT, ldv, ldk, ldP;
};

// Shared-memory layout of the K-tiled kernels (byte offsets).
struct KLds {
  int off_dO, off_dP, off_red, off_redo, off_a, off_b, off_bl, off_in, off_small, total;
};

// Value-slab width: 128 columns for bf16, 64 for fp32.
static int vs_for(const Shape &s) { return s.io == IO_BF16 ? 128 : 64; }

static KLds k_lds(const Shape &s, int n_in) {
  const int es = s.esz(), Cp = round_up(s.C, 32), VS = vs_for(s);
  const int ldv = VS + 32 / es, ldk = 32 + 32 / es, ldP = Cp + 4;
  KLds L;
  int off = Cp * ldv * es;          // V slab
  L.off_dO = off; off += Cp * ldv * es;
  L.off_dP = off; off += Cp * ldP * 4;
  L.off_red = off; off += 2 * s.C * 32 * 4;
  L.off_redo = off; off += s.C * 32 * 4;
  L.off_a = off; off += Cp * 36 * 4;  // fp32 gated operand for the sub-chunk products
  L.off_b = off; off += Cp * ldk * es;
  L.off_bl = off; off += (es == 2 ? Cp * ldk * es : 0);
  L.off_in = off; off += n_in * Cp * 32 * es;
  L.off_small = off; off += 640 * 4;
  L.total = off;
  return L;
}
static int n_in_dq(const Shape &) { return 2; }                           // log alpha, k
static int n_in_dk(const Shape &s) { return s.io == IO_BF16 ? 5 : 4; }  // q, k, log alpha, dq (+ lo)

// Small-buffer offsets inside the "small" region (floats).
enum { SM_TOT = 0, SM_G = 128, SM_GAM = 224, SM_RED = 256, SM_CARRY = 384, SM_BT = 416 };

// Operand pair for a product that reduces over 16 or 32 value columns of the
// transposed state: NVB2 = true takes two stacked 16x16 accumulators (32-deep
// step), false a single one (a 16-deep step; fp32 only, slots 4..7 unused).
// hi + lo = the fp32 state to ~16 mantissa bits for bf16; lo is unused for fp32.
template <typename T>
__device__ __forceinline__ void acc_frag_split(f4 a0, f4 a1, frag_t<T> &hi, frag_t<T> &lo) {
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

// A operand matching a single accumulator block: X[r0 + j][c0 + 4g + i], i < 4.
__device__ __forceinline__ f4 ld_row_perm_lo_f32(const float *X, int ld, int r0, int c0) {
  const int l = lane_id();
  return *(const f4 *)(X + (r0 + (l & 15)) * ld + c0 + 4 * (l >> 4));
}
__device__ __forceinline__ f4 mma_f32_x16(f4 c, f4 a, f4 b) {
#pragma unroll
  for (int i = 0; i < 4; ++i) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], c, 0, 0, 0);
  return c;
}

// acc[I][kb] += X[16I rows][value columns of this wave's blocks] * state^T, where
// X is the slab tile (dO for dq, V for dk) and st the wave's state blocks.
template <typename T, int NVB>
__device__ __forceinline__ void inter_product(f4 (&acc)[4][2], const T *X, int ldv, int nb, int w,
                                              f4 (&st)[NVB][2]) {
  if constexpr (NVB == 1) {
    const int l = lane_id();
    (void)l;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      for (int I = 0; I < nb; ++I)
          acc[I][kb] = mma_f32_x16(acc[I][kb], ld_row_perm_lo_f32((const float *)X, ldv, 16 * I, 16 * w),
                                   st[0][kb]);
  } else {
#pragma unroll
    for (int p = 0; p < NVB / 2; ++p)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        frag_t<T> bh, bl;
        acc_frag_split<T>(st[2 * p][kb], st[2 * p + 1][kb], bh, bl);
        for (int I = 0; I < nb; ++I) {
          const frag_t<T> af = ld_row_perm<T>(X, ldv, 16 * I, 16 * (w * NVB + 2 * p));
          acc[I][kb] = mma<T>(acc[I][kb], af, bh);
          if constexpr (sizeof(T) == 2) acc[I][kb] = mma<T>(acc[I][kb], af, bl);
        }
      }
  }
}

// st[m][kb] = gamma (.) st + Y^T B over the chunk (Y = V for S, dO for dS; B =
// the gated key/query operand with its bf16 residual), for this wave's blocks.
template <typename T, int NVB>
__device__ __forceinline__ void state_update(f4 (&st)[NVB][2], const T *Y, int ldv, const T *Bh,
                                             const T *Bl, int ldk, int Cp, int w, const float *gam) {
  const int j = lane_id() & 15;
  const float g0 = gam[j], g1 = gam[16 + j];
#pragma unroll
  for (int m = 0; m < NVB; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      st[m][0][r] *= g0;
      st[m][1][r] *= g1;
    }
  for (int s = 0; s < Cp / 32; ++s) {
    const frag_t<T> b0 = ld_col<T>(Bh, ldk, 32 * s, 0), b1 = ld_col<T>(Bh, ldk, 32 * s, 16);
    frag_t<T> l0, l1;
    if constexpr (sizeof(T) == 2) {
      l0 = ld_col<T>(Bl, ldk, 32 * s, 0);
      l1 = ld_col<T>(Bl, ldk, 32 * s, 16);
    }
#pragma unroll
    for (int m = 0; m < NVB; ++m) {
      const frag_t<T> ay = ld_col<T>(Y, ldv, 32 * s, 16 * (w * NVB + m));
      st[m][0] = mma<T>(st[m][0], ay, b0);
      st[m][1] = mma<T>(st[m][1], ay, b1);
      if constexpr (sizeof(T) == 2) {
        st[m][0] = mma<T>(st[m][0], ay, l0);
        st[m][1] = mma<T>(st[m][1], ay, l1);
      }
    }
  }
}

// fp32 fragments straight from fp32 LDS tiles: row orientation
// X[r0 + j][c0 + 8g + i] and column orientation X[r0 + 8g + i][c0 + j].
__device__ __forceinline__ f8 ldf_row(const float *X, int ld, int r0, int c0) {
  const int l = lane_id();
  const float *p = X + (r0 + (l & 15)) * ld + c0 + 8 * (l >> 4);
  const f4 a = *(const f4 *)p, b = *(const f4 *)(p + 4);
  return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}
__device__ __forceinline__ f8 ldf_col(const float *X, int ld, int r0, int c0) {
  const int l = lane_id();
  const float *p = X + (r0 + 8 * (l >> 4)) * ld + c0 + (l & 15);
  f8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = p[i * ld];
  return r;
}

// acc += a b for fp32 fragments: on bf16 hardware tiles each operand is split
// into hi + lo and the three significant cross terms are accumulated.
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

// Sum of the partials of the four waves (each over its value columns):
// waves 2, 3 publish, waves 0, 1 add theirs; the result is red[0] + red[1].
__device__ __forceinline__ void reduce_partials(f4 (&acc)[4][2], float *red, int nb, int C, int w,
                                                int g, int j) {
  if (w >= 2)
#pragma unroll
    for (int I = 0; I < 4; ++I)
      if (I < nb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) red[(w - 2) * C * 32 + (16 * I + 4 * g + r) * 32 + 16 * kb + j] = acc[I][kb][r];
  __syncthreads();
  if (w < 2)
#pragma unroll
    for (int I = 0; I < 4; ++I)
      if (I < nb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) red[w * C * 32 + (16 * I + 4 * g + r) * 32 + 16 * kb + j] += acc[I][kb][r];
  __syncthreads();
}

// Block-local cumsum of log alpha for factor thread (feature kk, block I).
template <typename T>
__device__ __forceinline__ float block_cumsum(const T *sLa, int I, int kk, float (&B)[16]) {
  float t = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    t += (float)sLa[(16 * I + r) * 32 + kk];
    B[r] = t;
  }
  return t;
}

// Per-chunk decay bookkeeping shared by the factor threads: publishes the block
// totals, then returns the log decay before this block (pre) and of the chunk (Bl),
// and writes the chunk decay gamma and the non-adjacent block factors to LDS.
__device__ __forceinline__ void block_decays(float *sm, int nb, int I, int kk, bool fv, float &pre,
                                             float &Bl) {
  pre = 0.f;
  Bl = 0.f;
  for (int I2 = 0; I2 < nb; ++I2) {
    const float t = sm[SM_TOT + I2 * 32 + kk];
    if (I2 < I) pre += t;
    Bl += t;
  }
  if (I == 2) sm[SM_G + kk] = __expf(sm[SM_TOT + 32 + kk]);
  if (I == 3) {
    sm[SM_G + 32 + kk] = __expf(sm[SM_TOT + 32 + kk] + sm[SM_TOT + 64 + kk]);
    sm[SM_G + 64 + kk] = __expf(sm[SM_TOT + 64 + kk]);
  }
  if (I == 0) sm[SM_GAM + kk] = fv ? __expf(Bl) : 0.f;
}

// ------------------------------------------------------------------ bwd_dq
template <typename T, int NVB, int NSLAB>
__global__ void __launch_bounds__(256) bwd_dq_kernel(KArgs a, KLds L) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr bool SPLIT = sizeof(T) == 2;
  constexpr int VS = NVB * 64, EV = 16 / sizeof(T);
  constexpr int NS = (64 * VS / EV + 255) / 256;
  constexpr int NI = (64 * 32 / EV + 255) / 256;
  int bh, kt;
  xcd_map(a.BH, a.KT, bh, kt);
  const int w = wave_id(), l = lane_id(), g = l >> 4, j = l & 15, tid = threadIdx.x;
  const int K = a.K, V = a.V, C = a.C, Cp = a.Cp, nb = C >> 4;
  const int ldv = a.ldv, ldk = a.ldk, ldP = a.ldP;
  const int k0 = kt * 32;
  T *sV = (T *)smem;
  T *sdO = (T *)(smem + L.off_dO);
  float *sdP = (float *)(smem + L.off_dP);
  float *sRed = (float *)(smem + L.off_red);
  float *sRedO = (float *)(smem + L.off_redo);
  float *sKs = (float *)(smem + L.off_a);
  T *sKt = (T *)(smem + L.off_b);
  T *sKtl = (T *)(smem + L.off_bl);
  T *sInLa = (T *)(smem + L.off_in), *sInK = sInLa + Cp * 32;
  float *sm = (float *)(smem + L.off_small);

  for (int i = tid; i < Cp * ldP; i += blockDim.x) sdP[i] = 0.f;
  for (int i = tid; i < Cp * 36; i += blockDim.x) sKs[i] = 0.f;
  for (int i = tid; i < Cp * ldk; i += blockDim.x) {
    sKt[i] = cvt<T>(0.f);
    if constexpr (SPLIT) sKtl[i] = cvt<T>(0.f);
  }

  f4 S[NSLAB][NVB][2];
#pragma unroll
  for (int sl = 0; sl < NSLAB; ++sl)
#pragma unroll
    for (int m = 0; m < NVB; ++m)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int vv = sl * VS + 16 * (w * NVB + m) + 4 * g + r, kq = k0 + 16 * kb + j;
          S[sl][m][kb][r] = (a.S0 && vv < V && kq < K) ? a.S0[((int64_t)bh * K + kq) * V + vv] : 0.f;
        }

  const T *kin = (const T *)a.k, *lain = (const T *)a.la, *vin = (const T *)a.v;
  const T *dOin = (const T *)a.dO;
  T *dqo = (T *)a.dq, *dqlo = (T *)a.dq_lo;
  const bool ft = tid < 32 * nb;  // factor thread: feature kk of row block Ib
  const int kk = tid & 31, Ib = tid >> 5, kf = k0 + kk;
  const bool fv = kf < K;
  const int nblk = nb * (nb + 1) / 2;

  TileRegs<T, NS> pV, pD;
  TileRegs<T, NI> pLa, pK;
  const int64_t hK = (int64_t)bh * a.T * K, hV = (int64_t)bh * a.T * V;  // head bases
  auto load_in = [&](int n) {
    const int rv = min(C, a.T - n * C);
    pLa.load(lain + hK + (n * C * K + k0), K, Cp, 32, rv, K - k0);
    pK.load(kin + hK + (n * C * K + k0), K, Cp, 32, rv, K - k0);
  };
  auto load_slab = [&](int n, int sl) {
    const int rv = min(C, a.T - n * C);
    pV.load(vin + hV + (n * C * V + sl * VS), V, Cp, VS, rv, V - sl * VS);
    pD.load(dOin + hV + (n * C * V + sl * VS), V, Cp, VS, rv, V - sl * VS);
  };
  __syncthreads();
  load_in(0);
  load_slab(0, 0);

  for (int n = 0; n < a.N; ++n) {
    const int t0 = n * C, rv = min(C, a.T - t0);
    const int64_t rb = (int64_t)bh * a.T + t0;
    // phase 0: gate factors; gated key operands for the products
    pLa.store(sInLa, 32, Cp, 32);
    pK.store(sInK, 32, Cp, 32);
    __syncthreads();
    if (ft) {
      float Bloc[16];
      sm[SM_TOT + Ib * 32 + kk] = block_cumsum(sInLa, Ib, kk, Bloc);
    }
    __syncthreads();
    if (ft) {
      float Bloc[16], pre, Bl;
      const float tot = block_cumsum(sInLa, Ib, kk, Bloc);
      block_decays(sm, nb, Ib, kk, fv, pre, Bl);
      const float ekt = __expf(Bl - pre - tot);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 16 * Ib + r;
        const float ks = (float)sInK[row * 32 + kk] * __expf(tot - Bloc[r]);
        sKs[row * 36 + kk] = ks;
        const float ktv = ks * ekt;
        const T hi = cvt<T>(ktv);
        sKt[row * ldk + kk] = hi;
        if constexpr (SPLIT) sKtl[row * ldk + kk] = cvt<T>(ktv - (float)hi);
      }
    }
    __syncthreads();

    // phase 1: dP, dq_inter (with S_[n]) and the state update, per value slab
    f4 accQ[4][2], accP[3];
#pragma unroll
    for (int I = 0; I < 4; ++I) accQ[I][0] = accQ[I][1] = zero4();
#pragma unroll
    for (int b = 0; b < 3; ++b) accP[b] = zero4();
#pragma unroll
    for (int sl = 0; sl < NSLAB; ++sl) {
      pV.store(sV, ldv, Cp, VS);
      pD.store(sdO, ldv, Cp, VS);
      __syncthreads();
      if (sl + 1 < NSLAB) load_slab(n, sl + 1);
      else if (n + 1 < a.N) load_slab(n + 1, 0);
#pragma unroll
      for (int bi = 0; bi < 3; ++bi) {
        const int b = w + 4 * bi;
        if (b < nblk) {
          int I, J;
          tri_block(b, I, J);
#pragma unroll
          for (int s = 0; s < VS / 32; ++s)
            accP[bi] = mma<T>(accP[bi], ld_row<T>(sdO, ldv, 16 * I, 32 * s), ld_row<T>(sV, ldv, 16 * J, 32 * s));
        }
      }
      inter_product<T, NVB>(accQ, sdO, ldv, nb, w, S[sl]);
      state_update<T, NVB>(S[sl], sV, ldv, sKt, sKtl, ldk, Cp, w, sm + SM_GAM);
      __syncthreads();
    }
    if (n + 1 < a.N) load_in(n + 1);

    // phase 2: publish dP, reduce the dq_inter partials
#pragma unroll
    for (int bi = 0; bi < 3; ++bi) {
      const int b = w + 4 * bi;
      if (b < nblk) {
        int I, J;
        tri_block(b, I, J);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 16 * I + 4 * g + r, cj = 16 * J + j;
          const float val = cj > row ? 0.f : accP[bi][r];
          sdP[row * ldP + cj] = val;
          if (kt == 0) a.dP[(((int64_t)bh * a.N + n) * C + row) * C + cj] = val;
        }
      }
    }
    if (kt == 0)  // blocks above the diagonal of the stored dP are zero
      for (int idx = tid; idx < C * C; idx += blockDim.x) {
        const int row = idx / C, cj = idx - row * C;
        if ((cj >> 4) > (row >> 4)) a.dP[((int64_t)bh * a.N + n) * C * C + idx] = 0.f;
      }
    reduce_partials(accQ, sRed, nb, C, w, g, j);

    // phase 3: orange dq blocks, sum over J < I of dP_IJ (ks_J (.) g_IJ)
    for (int t = w; t < 2 * (nb - 1); t += 4) {
      const int I = 1 + (t >> 1), kb = t & 1;
      f4 acc = zero4();
      for (int s = 0; s < (16 * I + 31) / 32; ++s) {
        const int J = 2 * s + (g >> 1);
        const float sc = J >= I ? 0.f : (J <= I - 2 ? sm[SM_G + pair_idx(I, J) * 32 + 16 * kb + j] : 1.f);
        f8 bf = ldf_col(sKs, 36, 32 * s, 16 * kb);
#pragma unroll
        for (int i = 0; i < 8; ++i) bf[i] *= sc;
        acc = mma_split3<T>(acc, ldf_row(sdP, ldP, 16 * I, 32 * s), bf);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sRedO[(16 * I + 4 * g + r) * 32 + 16 * kb + j] = acc[r];
    }
    __syncthreads();

    // phase 4: dq = Lambda (.) inter + intra (orange + diagonal block in fp32)
    if (ft) {
      float Bloc[16], pre, Bl;
      const float tot = block_cumsum(sInLa, Ib, kk, Bloc);
      pre = 0.f;
      for (int I2 = 0; I2 < Ib; ++I2) pre += sm[SM_TOT + I2 * 32 + kk];
      (void)Bl;
      const float ez = __expf(pre), eup = __expf(-tot);
      const bool wide = fv && (-tot > kWideRangeB);
      float kh[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float kv = (float)sInK[(16 * Ib + r) * 32 + kk];
        kh[r] = wide ? kv : kv * __expf(tot - Bloc[r]) * eup;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 16 * Ib + r;
        const float inter = sRed[row * 32 + kk] + sRed[C * 32 + row * 32 + kk];
        const float orange = Ib > 0 ? sRedO[row * 32 + kk] : 0.f;
        const float qf = __expf(Bloc[r]);
        float pink = 0.f, dq;
        const float *dprow = sdP + row * ldP + 16 * Ib;
        if (!wide) {
#pragma unroll
          for (int jj = 0; jj <= r; ++jj) pink += dprow[jj] * kh[jj];
          dq = qf * (ez * inter + orange + pink);
        } else {
#pragma unroll
          for (int jj = 0; jj <= r; ++jj) pink += dprow[jj] * kh[jj] * __expf(Bloc[r] - Bloc[jj]);
          dq = qf * (ez * inter + orange) + pink;
        }
        if (row < rv && fv) {
          const T hi = cvt<T>(dq);
          dqo[(rb + row) * K + kf] = hi;
          if constexpr (SPLIT) dqlo[(rb + row) * K + kf] = cvt<T>(dq - (float)hi);
        }
      }
    }
    __syncthreads();
  }

  // final-state term of the gate gradient: rowsum(S_T (.) dS_T) per feature
  if (a.dST) {
    float part[2] = {0.f, 0.f};
#pragma unroll
    for (int sl = 0; sl < NSLAB; ++sl)
#pragma unroll
      for (int m = 0; m < NVB; ++m)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int vv = sl * VS + 16 * (w * NVB + m) + 4 * g + r, kq = k0 + 16 * kb + j;
            if (vv < V && kq < K) part[kb] += S[sl][m][kb][r] * a.dST[((int64_t)bh * K + kq) * V + vv];
          }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      part[kb] += __shfl_xor(part[kb], 16);
      part[kb] += __shfl_xor(part[kb], 32);
    }
    if (g == 0) {
      sm[SM_RED + w * 32 + j] = part[0];
      sm[SM_RED + w * 32 + 16 + j] = part[1];
    }
    __syncthreads();
    if (tid < 32 && k0 + tid < K)
      a.cST[(int64_t)bh * K + k0 + tid] = sm[SM_RED + tid] + sm[SM_RED + 32 + tid] +
                                          sm[SM_RED + 64 + tid] + sm[SM_RED + 96 + tid];
  }
}

// ------------------------------------------------------------------ bwd_dk
template <typename T, int NVB, int NSLAB>
__global__ void __launch_bounds__(256) bwd_dk_kernel(KArgs a, KLds L) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr bool SPLIT = sizeof(T) == 2;
  constexpr int VS = NVB * 64, EV = 16 / sizeof(T);
  constexpr int NS = (64 * VS / EV + 255) / 256;
  constexpr int NI = (64 * 32 / EV + 255) / 256;
  constexpr int NP = 64 * 64 / 4 / 256;  // dP chunk (fp32) vectors per thread
  int bh, kt;
  xcd_map(a.BH, a.KT, bh, kt);
  const int w = wave_id(), l = lane_id(), g = l >> 4, j = l & 15, tid = threadIdx.x;
  const int K = a.K, V = a.V, C = a.C, Cp = a.Cp, nb = C >> 4;
  const int ldv = a.ldv, ldk = a.ldk, ldP = a.ldP;
  const int k0 = kt * 32;
  T *sV = (T *)smem;
  T *sdO = (T *)(smem + L.off_dO);
  float *sdP = (float *)(smem + L.off_dP);
  float *sRed = (float *)(smem + L.off_red);
  float *sRedO = (float *)(smem + L.off_redo);
  float *sQh = (float *)(smem + L.off_a);
  T *sQt = (T *)(smem + L.off_b);
  T *sQtl = (T *)(smem + L.off_bl);
  T *sInQ = (T *)(smem + L.off_in), *sInK = sInQ + Cp * 32, *sInLa = sInQ + 2 * Cp * 32;
  T *sInDq = sInQ + 3 * Cp * 32, *sInDql = sInQ + 4 * Cp * 32;
  float *sm = (float *)(smem + L.off_small);

  for (int i = tid; i < Cp * 36; i += blockDim.x) sQh[i] = 0.f;
  for (int i = tid; i < Cp * ldk; i += blockDim.x) {
    sQt[i] = cvt<T>(0.f);
    if constexpr (SPLIT) sQtl[i] = cvt<T>(0.f);
  }
  if (tid < 32) sm[SM_CARRY + tid] = (a.cST && k0 + tid < K) ? a.cST[(int64_t)bh * K + k0 + tid] : 0.f;

  f4 dS[NSLAB][NVB][2];
#pragma unroll
  for (int sl = 0; sl < NSLAB; ++sl)
#pragma unroll
    for (int m = 0; m < NVB; ++m)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int vv = sl * VS + 16 * (w * NVB + m) + 4 * g + r, kq = k0 + 16 * kb + j;
          dS[sl][m][kb][r] = (a.dST && vv < V && kq < K) ? a.dST[((int64_t)bh * K + kq) * V + vv] : 0.f;
        }

  const T *qin = (const T *)a.q, *kin = (const T *)a.k, *lain = (const T *)a.la;
  const T *vin = (const T *)a.v, *dOin = (const T *)a.dO, *dqin = (const T *)a.dq_in;
  const T *dqlin = (const T *)a.dq_lo_in;
  T *dko = (T *)a.dk, *dlao = (T *)a.dla;
  const bool ft = tid < 32 * nb;
  const int kk = tid & 31, Jb = tid >> 5, kf = k0 + kk;
  const bool fv = kf < K;

  TileRegs<T, NS> pV, pD;
  TileRegs<T, NI> pQ, pK, pLa, pDq, pDql;
  TileRegs<float, NP> pP;
  const int64_t hK = (int64_t)bh * a.T * K, hV = (int64_t)bh * a.T * V;  // head bases
  const float *dPh = a.dP + (int64_t)bh * a.N * C * C;
  auto load_in = [&](int n) {
    const int rv = min(C, a.T - n * C);
    const int off = n * C * K + k0;
    pQ.load(qin + hK + off, K, Cp, 32, rv, K - k0);
    pK.load(kin + hK + off, K, Cp, 32, rv, K - k0);
    pLa.load(lain + hK + off, K, Cp, 32, rv, K - k0);
    pDq.load(dqin + hK + off, K, Cp, 32, rv, K - k0);
    if constexpr (SPLIT) pDql.load(dqlin + hK + off, K, Cp, 32, rv, K - k0);
    pP.load(dPh + n * C * C, C, Cp, Cp, C, C);
  };
  auto load_slab = [&](int n, int sl) {
    const int rv = min(C, a.T - n * C);
    pV.load(vin + hV + (n * C * V + sl * VS), V, Cp, VS, rv, V - sl * VS);
    pD.load(dOin + hV + (n * C * V + sl * VS), V, Cp, VS, rv, V - sl * VS);
  };
  __syncthreads();
  load_in(a.N - 1);
  load_slab(a.N - 1, 0);

  for (int n = a.N - 1; n >= 0; --n) {
    const int t0 = n * C, rv = min(C, a.T - t0);
    const int64_t rb = (int64_t)bh * a.T + t0;
    // phase 0: gate factors and the query-side operands of this workgroup's features
    pQ.store(sInQ, 32, Cp, 32);
    pK.store(sInK, 32, Cp, 32);
    pLa.store(sInLa, 32, Cp, 32);
    pDq.store(sInDq, 32, Cp, 32);
    if constexpr (SPLIT) pDql.store(sInDql, 32, Cp, 32);
    pP.store(sdP, ldP, Cp, Cp);
    __syncthreads();
    if (ft) {
      float Bloc[16];
      sm[SM_TOT + Jb * 32 + kk] = block_cumsum(sInLa, Jb, kk, Bloc);
    }
    __syncthreads();
    if (ft) {
      float Bloc[16], pre, Bl;
      const float tot = block_cumsum(sInLa, Jb, kk, Bloc);
      block_decays(sm, nb, Jb, kk, fv, pre, Bl);
      const float ez = __expf(pre);
      (void)tot;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 16 * Jb + r;
        const float qhv = (float)sInQ[row * 32 + kk] * __expf(Bloc[r]);
        sQh[row * 36 + kk] = qhv;
        const float qt = qhv * ez;
        const T hi = cvt<T>(qt);
        sQt[row * ldk + kk] = hi;
        if constexpr (SPLIT) sQtl[row * ldk + kk] = cvt<T>(qt - (float)hi);
      }
    }
    __syncthreads();

    // phase 1: dk_inter with dS_[n+1], then dS_[n], per value slab
    f4 accK[4][2];
#pragma unroll
    for (int J = 0; J < 4; ++J) accK[J][0] = accK[J][1] = zero4();
#pragma unroll
    for (int sl = 0; sl < NSLAB; ++sl) {
      pV.store(sV, ldv, Cp, VS);
      pD.store(sdO, ldv, Cp, VS);
      __syncthreads();
      if (sl + 1 < NSLAB) load_slab(n, sl + 1);
      else if (n > 0) load_slab(n - 1, 0);
      inter_product<T, NVB>(accK, sV, ldv, nb, w, dS[sl]);
      state_update<T, NVB>(dS[sl], sdO, ldv, sQt, sQtl, ldk, Cp, w, sm + SM_GAM);
      __syncthreads();
    }
    if (n > 0) load_in(n - 1);
    reduce_partials(accK, sRed, nb, C, w, g, j);

    // phase 3: orange dk blocks, sum over I > J of dP_IJ^T (qh_I (.) g_IJ)
    for (int t = w; t < 2 * (nb - 1); t += 4) {
      const int J = t >> 1, kb = t & 1;
      f4 acc = zero4();
      for (int s = (16 * (J + 1)) / 32; s < Cp / 32; ++s) {
        const int I = 2 * s + (g >> 1);
        const float sc = I <= J ? 0.f : (I >= J + 2 ? sm[SM_G + pair_idx(I, J) * 32 + 16 * kb + j] : 1.f);
        f8 bf = ldf_col(sQh, 36, 32 * s, 16 * kb);
#pragma unroll
        for (int i = 0; i < 8; ++i) bf[i] *= sc;
        acc = mma_split3<T>(acc, ldf_col(sdP, ldP, 32 * s, 16 * J), bf);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) sRedO[(16 * J + 4 * g + r) * 32 + 16 * kb + j] = acc[r];
    }
    __syncthreads();

    // phase 4: dk, dA = q dq - k dk, reverse cumulative sum -> dlog alpha
    float dA[16];
    if (ft) {
      float Bloc[16], pre = 0.f;
      const float tot = block_cumsum(sInLa, Jb, kk, Bloc);
      float Bl = 0.f;
      for (int I2 = 0; I2 < nb; ++I2) {
        const float t = sm[SM_TOT + I2 * 32 + kk];
        if (I2 < Jb) pre += t;
        Bl += t;
      }
      const float ekt = __expf(Bl - pre - tot), eup = __expf(-tot);
      const bool wide = fv && (-tot > kWideRangeB);
      float qh[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float q = (float)sInQ[(16 * Jb + r) * 32 + kk];
        qh[r] = wide ? q : q * __expf(Bloc[r]);
      }
      // diagonal block in fp32: pink[r] = sum_{i >= r} dP[i][r] q[i] exp(B_i - B_r)
      // (factorised: pink[r] is scaled by exp(tot - B_r) below; the wide
      // fallback forms each pairwise decay and is added unscaled)
      float pink[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) pink[r] = 0.f;
      const float *dpb = sdP + 16 * Jb * ldP + 16 * Jb;
      if (!wide) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
          for (int r = 0; r <= i; ++r) pink[r] += dpb[i * ldP + r] * qh[i];
#pragma unroll
        for (int r = 0; r < 16; ++r) pink[r] *= eup;
      } else {
#pragma unroll 1
        for (int r = 0; r < 16; ++r) {
          float s = 0.f;
          for (int i = r; i < 16; ++i) s += dpb[i * ldP + r] * qh[i] * __expf(Bloc[i] - Bloc[r]);
          pink[r] = s;
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 16 * Jb + r;
        const float inter = sRed[row * 32 + kk] + sRed[C * 32 + row * 32 + kk];
        const float orange = Jb < nb - 1 ? sRedO[row * 32 + kk] : 0.f;
        const float kfr = __expf(tot - Bloc[r]);
        const float dk = wide ? kfr * (ekt * inter + orange) + pink[r]
                              : kfr * (ekt * inter + orange + pink[r]);
        float dqv = (float)sInDq[row * 32 + kk];
        if constexpr (SPLIT) dqv += (float)sInDql[row * 32 + kk];
        dA[r] = (float)sInQ[row * 32 + kk] * dqv - (float)sInK[row * 32 + kk] * dk;
        if (row < rv && fv) dko[(rb + row) * K + kf] = cvt<T>(dk);
      }
      float s = 0.f;
#pragma unroll
      for (int r = 15; r >= 0; --r) {
        s += dA[r];
        dA[r] = s;
      }
      sm[SM_BT + Jb * 32 + kk] = s;
    }
    __syncthreads();
    if (ft) {
      float later = sm[SM_CARRY + kk];
      for (int J2 = Jb + 1; J2 < nb; ++J2) later += sm[SM_BT + J2 * 32 + kk];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 16 * Jb + r;
        if (row < rv && fv) dlao[(rb + row) * K + kf] = cvt<T>(dA[r] + later);
      }
    }
    __syncthreads();
    if (tid < 32) {
      float c = sm[SM_CARRY + tid];
      for (int J2 = 0; J2 < nb; ++J2) c += sm[SM_BT + J2 * 32 + tid];
      sm[SM_CARRY + tid] = c;
    }
  }
}

// ------------------------------------------------------------------ launchers

size_t lds_bwd_dq(const Shape &s) { return (size_t)k_lds(s, n_in_dq(s)).total; }
size_t lds_bwd_dk(const Shape &s) { return (size_t)k_lds(s, n_in_dk(s)).total; }

template <typename Kern, typename... Args>
static hipError_t launch_generic(Kern kern, dim3 grid, dim3 block, size_t lds, hipStream_t st,
                                 bool &attr, Args... args) {
  if (!attr) {
    hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr = true;
  }
  hipLaunchKernelGGL(kern, grid, block, lds, st, args...);
  return hipGetLastError();
}

static KArgs make_kargs(const Shape &s) {
  KArgs a{};
  a.BH = s.BH; a.T = s.T; a.K = s.K; a.V = s.V; a.C = s.C; a.N = s.N;
  a.Cp = round_up(s.C, 32);
  a.KT = (s.K + 31) / 32;
  a.ldv = vs_for(s) + 32 / s.esz();
  a.ldk = 32 + 32 / s.esz();
  a.ldP = a.Cp + 4;
  return a;
}

template <typename T, int NVB, int NSLAB>
static hipError_t run_dq(const KArgs &a, const KLds &L, hipStream_t st) {
  static bool attr = false;
  return launch_generic(bwd_dq_kernel<T, NVB, NSLAB>, dim3(a.BH * a.KT), dim3(256), L.total, st,
                        attr, a, L);
}
template <typename T, int NVB, int NSLAB>
static hipError_t run_dk(const KArgs &a, const KLds &L, hipStream_t st) {
  static bool attr = false;
  return launch_generic(bwd_dk_kernel<T, NVB, NSLAB>, dim3(a.BH * a.KT), dim3(256), L.total, st,
                        attr, a, L);
}

// Slab counts are rounded up to a power of two; extra slabs are all-zero.
template <bool DQ>
static hipError_t run_k(const Shape &s, const KArgs &a, const KLds &L, hipStream_t st) {
  const int VS = vs_for(s), nsl = (s.V + VS - 1) / VS;
#define GLA_RUN(T, NVB, NS) return DQ ? run_dq<T, NVB, NS>(a, L, st) : run_dk<T, NVB, NS>(a, L, st)
  if (s.io == IO_BF16) {
    if (nsl <= 1) GLA_RUN(bf16, 2, 1);
    if (nsl <= 2) GLA_RUN(bf16, 2, 2);
    if (nsl <= 4) GLA_RUN(bf16, 2, 4);
    GLA_RUN(bf16, 2, 8);
  }
  if (nsl <= 1) GLA_RUN(float, 1, 1);
  if (nsl <= 2) GLA_RUN(float, 1, 2);
  if (nsl <= 4) GLA_RUN(float, 1, 4);
  if (nsl <= 8) GLA_RUN(float, 1, 8);
  GLA_RUN(float, 1, 16);
#undef GLA_RUN
}

hipError_t launch_bwd_dq(const Shape &s, const void *k, const void *la, const void *v,
                         const float *S0, const void *dO, const float *dST, void *dq,
                         const Work &w, hipStream_t st) {
  KArgs a = make_kargs(s);
  a.k = k; a.la = la; a.v = v; a.dO = dO; a.S0 = S0; a.dST = dST; a.dq = dq; a.dq_lo = w.dq_lo;
  a.dP = w.dP; a.cST = w.cST;
  return run_k<true>(s, a, k_lds(s, n_in_dq(s)), st);
}

hipError_t launch_bwd_dk(const Shape &s, const void *q, const void *k, const void *la,
                         const void *v, const void *dO, const float *dST, const void *dq,
                         void *dk, void *dla, const Work &w, hipStream_t st) {
  KArgs a = make_kargs(s);
  a.q = q; a.k = k; a.la = la; a.v = v; a.dO = dO; a.dST = dST; a.dq_in = dq; a.dq_lo_in = w.dq_lo;
  a.dk = dk; a.dla = dla; a.dP = w.dP; a.cST = dST ? w.cST : nullptr;
  return run_k<false>(s, a, k_lds(s, n_in_dk(s)), st);
}

}  // namespace gla
