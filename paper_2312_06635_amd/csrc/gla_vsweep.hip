// gla_vsweep.hip -- the two sweeps over chunks that tile the value columns:
//
//   forward state pass (Sec. 4.2; the non-materialised pass of Sec. 3.3 and
//   App. B, Alg. 5), chunks n = 0 .. N-1:
//       O_n     = (Q (.) Lambda)_n S_[n] + P_n V_n
//       S_[n+1] = Diag(gamma_n) S_[n] + (K (.) Gamma)_n^T V_n
//   backward dv pass (App. B, Alg. 4/6 as corrected: the dS recurrence uses
//   Q (.) Lambda), chunks n = N-1 .. 0:
//       dV_n    = (K (.) Gamma)_n dS_[n+1] + P_n^T dO_n
//       dS_[n]  = Diag(gamma_n) dS_[n+1] + (Q (.) Lambda)_n^T dO_n
//
// Both have the same shape: a state R (S or dS, d_k x d_v, fp32) carried
// across chunks, an output X_n R + intra, and an update R <- gamma R + Y_n^T Z_n.
// The columns of R evolve independently (the gate of Eq. 3 scales rows), so a
// workgroup owns a 64-column tile of one head for the whole sequence and no
// state crosses workgroups.
//
// Workgroup = 8 waves.  Wave w owns value columns 16 (w & 3) .. +16 of the tile
// and key features [ (w >> 2) KP/2, (w >> 2 + 1) KP/2 ) of R, held as fp32
// matrix-core accumulators.  The output contraction over key features is thus
// split between the two halves: the upper half hands its partial to the lower
// half through LDS, and the lower half adds the intra-chunk term and writes
// the output.
//
// Key-feature order inside the accumulators: accumulator pair (2s, 2s+1) of a
// lane in group g holds features 32 s + 8 g + (0..7), so the pair is directly
// the A operand of the next output product, whose B operand is then one
// contiguous 16-byte LDS read.  The update's transposed operand is read with
// LDS transpose reads pointed at the matching permuted columns (ld_col_perm).
//
// The output is computed transposed (value columns x time), so each lane ends
// with four consecutive value columns of one time row: one 8-byte (bf16) or
// 16-byte (fp32) store.
//
// Tiles of chunk n+2 are fetched with buffer loads into one of two register
// sets while chunk n computes; each lane's byte offsets are fixed for the
// whole sweep (rows past the sequence end fall outside the buffer's range and
// read as zero).
//
// Value-side gate (the general form G_t = alpha_t^T beta_t of App. C): with
// E = the chunk-local inclusive cumsum of log beta per value column (computed
// here, per chunk, in LDS), Vh = V (.) exp(-E) and Oh = dO (.) exp(E),
//       O_n     = exp(E) (.) ((Q (.) Lambda)_n S_[n] + P_n Vh_n)
//       S_[n+1] = (Diag(gamma_n) S_[n] + (K (.) Gamma)_n^T Vh_n) Diag(exp(E_last))
//       dV_n    = exp(-E) (.) ((K (.) Gamma)_n D + P_n^T Oh_n),  D = dS_[n+1] Diag(exp(E_last))
//       dS_[n]  = Diag(gamma_n) D + (Q (.) Lambda)_n^T Oh_n,
// which is exact; exp(-E) grows with the decay range of beta inside one chunk,
// so that range must stay below ~80 (fp32 exponent), e.g. by a shorter chunk.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

constexpr int kThreads = 512;
constexpr int kTile = 64;  // value columns per workgroup

static int pow2_at_least(int x, int lo) {
  int p = lo;
  while (p < x) p *= 2;
  return p;
}

struct SweepArgs {
  const void *X, *Y, *Z, *P;  // X: output operand, Y: update operand, Z: value tile source
  const float *gam;
  const float *R0;  // initial state (nullable)
  const void *LB;   // log beta [BH][T][V] (value-side gate; the GB variant only)
  void *out;
  float *RN;        // final state (nullable)
  int BH, T, K, V, C, N, ntiles;
};

template <typename T> struct Pads;
template <> struct Pads<bf16> {
  // Row strides chosen so that 16-byte row reads (X, P) and transpose reads
  // (Y, Z) of a wave's 16-lane phase touch distinct LDS banks.
  static constexpr int row = 8, col = 32;
};
template <> struct Pads<float> {
  static constexpr int row = 4, col = 4;
};

template <typename T, int KP, int CP> struct SweepLayout {
  static constexpr int LDX = KP + Pads<T>::row;
  static constexpr int LDY = KP + Pads<T>::col;
  static constexpr int LDZ = kTile + Pads<T>::col;
  static constexpr int LDP = CP + Pads<T>::row;
  static constexpr int NI = CP / 16;
  static constexpr size_t offX = 0;
  static constexpr size_t offY = offX + sizeof(T) * CP * LDX;
  static constexpr size_t offZ = offY + sizeof(T) * CP * LDY;
  static constexpr size_t offP = offZ + sizeof(T) * CP * LDZ;
  static constexpr size_t offG = offP + sizeof(T) * CP * LDP;
  static constexpr size_t offO = offG + sizeof(float) * KP;
  static constexpr size_t total = offO + sizeof(f4) * 4 * NI * 64;
  // value-side gate: log beta tile, its chunk-local cumsum E, scan partials
  static constexpr int LDE = kTile + 4;
  static constexpr size_t offLB = total;
  static constexpr size_t offE = offLB + sizeof(T) * CP * LDZ;
  static constexpr size_t offScan = offE + sizeof(float) * CP * LDE;
  static constexpr size_t total_gb = offScan + sizeof(float) * 8 * kTile;
};

// Fragment whose reduction index runs down a column, like ld_col, but with the
// 16 columns taken in the permuted key-feature order of the state
// accumulators: lane (g, j) gets X[r0 + 8g + i][c0 + 8 (j / 4) + 4 h + j % 4].
// For bf16 each transpose read returns, to lane j of a 16-lane group, element
// j % 4 of the 4-vector loaded by lane 4 m + j / 4 (m = 0..3), so lane 4a + b
// points at row r0 + 8g + a, column c0 + 8 b + 4 h.
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

// bf16 tiles read with transpose loads (the update's key tile Y, the value
// tile Z and, backward, P) are stored with their 8-byte units XOR-permuted per
// row instead of padded.  A 32-lane phase of those loads touches rows
// 8g + 0..3 (g = 0, 1) of a 32-row block, four lanes per row, and with any
// padded stride rows r and r + 8 share LDS banks (a 2-way conflict on every
// load).  The permutations below give the eight rows disjoint banks; they use
// row bits 0, 1 and 3 only, so the second load of a fragment (rows + 4) and
// every 32-row block reuse the lane's base.  Stores stay conflict-free: each
// row's units are only permuted among themselves.
//   key rows of 2 KP bytes: unit u of row r at u ^ swz_key(r)
//   value / P rows of 128 (64) bytes: unit u at u ^ swz_val(r)
template <int KP> __device__ __forceinline__ int swz_key(int r) {
  if constexpr (KP >= 128) return (r & 1) | ((r & 2) << 2) | ((r & 8) << 1);
  else return ((r & 2) >> 1) | (r & 8);  // 128-byte rows: odd rows already use the other bank half
}
template <int RB> __device__ __forceinline__ int swz_val(int r) {
  if constexpr (RB >= 128) return ((r & 2) << 1) | (r & 8);
  else return (r & 8) >> 1;
}

// Transposed fragment (the ld_col / ld_col_perm element order) from such a
// tile: rb = row bytes, lb = the lane's base offset for a block starting at
// row 0 and column 0 (the column start c0 is XORed in).
__device__ __forceinline__ bf16x8 ld_tr_xor8(const bf16 *X, int rb, int r0, int c0, int lb) {
  const char *p = (const char *)X + r0 * rb + (lb ^ (2 * c0));
  s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)p);
  s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p + 4 * rb));
  return __builtin_bit_cast(bf16x8, s8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]});
}

// GB: value-side gate.
template <typename T, int KP, int CP, bool REV, bool GB>
__global__ void __launch_bounds__(kThreads) sweep_kernel(SweepArgs a) {
  using L = SweepLayout<T, KP, CP>;
  constexpr int KH = KP / 2;     // key features per wave half
  constexpr int NKB = KH / 16;   // state accumulators per wave
  constexpr int NS = KH / 32;    // 32-feature steps of the output contraction
  constexpr int NI = CP / 16;    // 16-row time blocks of a chunk
  constexpr int NSC = CP / 32;   // 32-row time steps of the update
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T *sX = (T *)(smem + L::offX);
  T *sY = (T *)(smem + L::offY);
  T *sZ = (T *)(smem + L::offZ);
  T *sP = (T *)(smem + L::offP);
  float *sG = (float *)(smem + L::offG);
  f4 *sO = (f4 *)(smem + L::offO);
  T *sLB = (T *)(smem + L::offLB);
  float *sE = (float *)(smem + L::offE), *sScan = (float *)(smem + L::offScan);

  int bh, tile;
  xcd_map(a.BH, a.ntiles, bh, tile);
  const int w = wave_id(), l = lane_id(), g = l >> 4, j = l & 15;
  const int cg = w & 3, kh = w >> 2;
  const int K = a.K, V = a.V, C = a.C, N = a.N;
  const int v0 = tile * kTile;
  const int cbase = 16 * cg;                // first column of this wave, tile-local
  const bool active = v0 + cbase < V;       // V is a multiple of 16
  const int fbase = kh * KH;
  const int col = v0 + cbase + j;
  // bf16 transposed-read lane bases (see swz_key / swz_val): row 8g + j/4 of
  // the block, four lanes per row
  constexpr bool XS = sizeof(T) == 2;
  constexpr int RBY = 2 * KP, RBZ = 2 * kTile, RBP = 2 * CP;
  const int Rl = 8 * g + (j >> 2), bq = j & 3;
  const int lbY0 = Rl * RBY + 8 * ((2 * bq) ^ swz_key<KP>(Rl)), lbY1 = Rl * RBY + 8 * ((2 * bq + 1) ^ swz_key<KP>(Rl));
  const int lbZ = Rl * RBZ + ((8 * bq) | (8 * swz_val<RBZ>(Rl)));
  const int lbP = Rl * RBP + ((8 * bq) | (8 * swz_val<RBP>(Rl)));
  auto col_z = [&](int r0, int c0) -> frag_t<T> {  // ld_col(sZ)
    if constexpr (XS) return ld_tr_xor8(sZ, RBZ, r0, c0, lbZ);
    else return ld_col<T>(sZ, L::LDZ, r0, c0);
  };
  auto zel = [&](int row, int c) {  // element (row, c) of the value tile
    if constexpr (XS) return row * kTile + (c ^ (swz_val<RBZ>(row) << 2));
    else return row * L::LDZ + c;
  };

  // ---- state
  f4 R[NKB];
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int f = fbase + 32 * (kb >> 1) + 8 * g + 4 * (kb & 1) + r;
      R[kb][r] = (a.R0 && active && f < K) ? a.R0[((int64_t)bh * K + f) * V + col] : 0.f;
    }

  // ---- tile loaders (per-lane offsets fixed for the sweep); two register
  // sets, so the tiles of chunk it+2 are in flight while chunk it computes
  struct Stage {
    TileLd<T, CP, KP, kThreads> x, y;
    TileLd<T, CP, kTile, kThreads> z, b;  // b: log beta (GB)
    TileLd<T, CP, CP, kThreads> p;
    float g;
  };
  Stage st0, st1;
  st0.x.init(K, C, K);
  st0.y.init(K, C, K);
  st0.z.init(V, C, V - v0);
  st0.p.init(C, C, C);
  if constexpr (GB) st0.b = st0.z;
  st1.x = st0.x;
  st1.y = st0.y;
  st1.z = st0.z;
  st1.p = st0.p;
  if constexpr (GB) st1.b = st0.z;
  const int esz = sizeof(T);
  const uint32_t goff = (int)threadIdx.x < K ? 4u * threadIdx.x : 0x80000000u;  // gamma: lanes past K read 0
  const T *Xh = (const T *)a.X + (int64_t)bh * a.T * K;
  const T *Yh = (const T *)a.Y + (int64_t)bh * a.T * K;
  const T *Zh = (const T *)a.Z + (int64_t)bh * a.T * V + v0;
  const T *LBh = GB ? (const T *)a.LB + (int64_t)bh * a.T * V + v0 : Zh;
  const T *Ph = (const T *)a.P + (int64_t)bh * N * C * C;
  const float *Gh = a.gam + (int64_t)bh * N * K;
  auto chunk_of = [&](int it) { return REV ? N - 1 - it : it; };
  // part 0: X tile, 1: Y tile, 2: value tile, 3: P tile and gamma
  auto fetch_part = [&](Stage &S, int n, int part) {
    const int t0 = n * C;
    const uint32_t remK = rsrc_bytes((int64_t)(a.T - t0) * K * esz);
    if (part == 0) S.x.load(make_rsrc(Xh + (int64_t)t0 * K, remK));
    if (part == 1) S.y.load(make_rsrc(Yh + (int64_t)t0 * K, remK));
    if (part == 2) {
      const uint32_t remV = rsrc_bytes(((int64_t)(a.T - t0) * V - v0) * esz);
      S.z.load(make_rsrc(Zh + (int64_t)t0 * V, remV));
      if constexpr (GB) S.b.load(make_rsrc(LBh + (int64_t)t0 * V, remV));
    }
    if (part == 3) {
      S.p.load(make_rsrc(Ph + (int64_t)n * C * C, (uint32_t)(C * C * esz)));
      S.g = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(make_rsrc(Gh + (int64_t)n * K, (uint32_t)(K * 4)), goff, 0, 0));
    }
  };
  auto fetch = [&](Stage &S, int n) {
#pragma unroll
    for (int part = 0; part < 4; ++part) fetch_part(S, n, part);
  };

  T *outh = (T *)a.out + (int64_t)bh * a.T * V;
  auto body = [&](Stage &S, int it) {
    const int n = chunk_of(it);
    const int t0 = n * C, rv = min(C, a.T - t0);
    S.x.store(sX, L::LDX);
    if constexpr (XS) {
      S.y.store_xor8(sY, KP, [](int r) { return swz_key<KP>(r); });
      S.z.store_xor8(sZ, kTile, [](int r) { return swz_val<RBZ>(r); });
      if constexpr (REV) S.p.store_xor8(sP, CP, [](int r) { return swz_val<RBP>(r); });
      else S.p.store(sP, L::LDP);  // read by rows (forward), padded
    } else {
      S.y.store(sY, L::LDY);
      S.z.store(sZ, L::LDZ);
      S.p.store(sP, L::LDP);
    }
    if constexpr (GB) S.b.store(sLB, L::LDZ);
    if ((int)threadIdx.x < KP) sG[threadIdx.x] = S.g;
    __syncthreads();
    if constexpr (GB) {
      // E = inclusive cumsum of log beta down each column (thread: column c,
      // rows RG grp .. +RG-1), then the value tile becomes Vh = V (.) exp(-E)
      // (forward) or Oh = dO (.) exp(E) (backward) in place.  Rows past the
      // chunk or the sequence read log beta = 0.
      constexpr int RG = CP / 8;
      const int c = threadIdx.x & (kTile - 1), grp = threadIdx.x / kTile;
      float part = 0.f;
#pragma unroll
      for (int r = 0; r < RG; ++r) part += (float)sLB[(grp * RG + r) * L::LDZ + c];
      sScan[grp * kTile + c] = part;
      __syncthreads();
      float pre = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < 8; ++g2)
        if (g2 < grp) pre += sScan[g2 * kTile + c];
#pragma unroll
      for (int r = 0; r < RG; ++r) {
        const int row = grp * RG + r;
        pre += (float)sLB[row * L::LDZ + c];
        sE[row * L::LDE + c] = pre;
        sZ[zel(row, c)] = cvt<T>((float)sZ[zel(row, c)] * __expf(REV ? pre : -pre));
      }
      __syncthreads();
      if constexpr (REV) {
        // D = dS_[n+1] Diag(exp(E_last)) before the chunk's products
        const float gb = __expf(sE[(CP - 1) * L::LDE + cbase + j]);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) R[kb] *= gb;
      }
    }

    // output, transposed: acc[I] = R^T X^T over this wave's key features (a
    // wave past the last value column computes zeros).  The loads of chunk
    // it + 2 are issued a quarter at a time between these products, so the
    // memory pipeline drains while the matrix cores work.
    const int nf = chunk_of(min(it + 2, N - 1));
    f4 acc[NI];
#pragma unroll
    for (int I = 0; I < NI; ++I) acc[I] = zero4();
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const frag_t<T> ra = acc_frag<T>(R[2 * s], R[2 * s + 1]);
#pragma unroll
      for (int I = 0; I < NI; ++I) acc[I] = mma<T>(acc[I], ra, ld_row<T>(sX, L::LDX, 16 * I, fbase + 32 * s));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int part = s * 4 / NS; part < (s + 1) * 4 / NS; ++part) fetch_part(S, nf, part);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (active) {
      if (kh == 0) {
        // intra-chunk term: O += P V (forward) or dV += P^T dO (backward)
#pragma unroll
        for (int I = 0; I < NI; ++I) {
          if constexpr (!REV) {
#pragma unroll
            for (int sc = 0; sc <= (16 * I + 15) / 32; ++sc)
              acc[I] = mma<T>(acc[I], col_z(32 * sc, cbase), ld_row<T>(sP, L::LDP, 16 * I, 32 * sc));
          } else {
#pragma unroll
            for (int sc = (16 * I) / 32; sc < NSC; ++sc)
            {
              frag_t<T> pf;
              if constexpr (XS) pf = ld_tr_xor8(sP, RBP, 32 * sc, 16 * I, lbP);
              else pf = ld_col<T>(sP, L::LDP, 32 * sc, 16 * I);
              acc[I] = mma<T>(acc[I], col_z(32 * sc, cbase), pf);
            }
          }
        }
      } else {
#pragma unroll
        for (int I = 0; I < NI; ++I) sO[(cg * NI + I) * 64 + l] = acc[I];
      }
      // state update: R <- gamma R + Y^T Z (then, with the value-side gate,
      // times the chunk decay exp(E_last) of this lane's value column)
      frag_t<T> zf[NSC];
#pragma unroll
      for (int sc = 0; sc < NSC; ++sc) zf[sc] = col_z(32 * sc, cbase);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int c0 = fbase + 32 * (kb >> 1);
        const f4 gm = *(const f4 *)(sG + c0 + 8 * g + 4 * (kb & 1));
        R[kb] *= gm;
#pragma unroll
        for (int sc = 0; sc < NSC; ++sc)
        {
          frag_t<T> yf;
          if constexpr (XS) yf = ld_tr_xor8(sY, RBY, 32 * sc, c0, (kb & 1) ? lbY1 : lbY0);
          else yf = ld_col_perm<T>(sY, L::LDY, 32 * sc, c0, kb & 1);
          R[kb] = mma<T>(R[kb], yf, zf[sc]);
        }
      }
      if constexpr (GB && !REV) {
        const float gb = __expf(sE[(CP - 1) * L::LDE + cbase + j]);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) R[kb] *= gb;
      }
    }
    __syncthreads();
    if (active && kh == 0) {
#pragma unroll
      for (int I = 0; I < NI; ++I) {
        f4 o = acc[I] + sO[(cg * NI + I) * 64 + l];
        const int row = 16 * I + j;
        if constexpr (GB) {
          const f4 e = *(const f4 *)(sE + row * L::LDE + cbase + 4 * g);
#pragma unroll
          for (int r = 0; r < 4; ++r) o[r] *= __expf(REV ? -e[r] : e[r]);
        }
        if (row < rv) {
          T *dst = outh + (int64_t)(t0 + row) * V + v0 + cbase + 4 * g;
          if constexpr (sizeof(T) == 2) {
            bf16x4 ov = bf16x4{(bf16)o[0], (bf16)o[1], (bf16)o[2], (bf16)o[3]};
            *(bf16x4 *)dst = ov;
          } else {
            *(f4 *)dst = o;
          }
        }
      }
    }
  };
  fetch(st0, chunk_of(0));
  if (N > 1) fetch(st1, chunk_of(1));
  for (int it = 0; it < N; it += 2) {
    body(st0, it);
    if (it + 1 < N) body(st1, it + 1);
  }
  if (a.RN && active) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int f = fbase + 32 * (kb >> 1) + 8 * g + 4 * (kb & 1) + r;
        if (f < K) a.RN[((int64_t)bh * K + f) * V + col] = R[kb][r];
      }
  }
}

int sweep_kp(const Shape &s) { return pow2_at_least(s.K, 64); }
int sweep_cp(const Shape &s) { return s.C <= 32 ? 32 : 64; }

template <typename T, int KP, int CP>
size_t sweep_lds() { return SweepLayout<T, KP, CP>::total_gb; }  // the larger, value-gate layout

size_t sweep_lds(const Shape &s) {
  const int KP = sweep_kp(s), CP = sweep_cp(s);
  if (KP > 256 || s.C > 64) return 0;
  const bool b = s.io == IO_BF16;
  if (!b && KP > 128) return 0;
#define GLA_LDS_CASE(kp, cp) \
  if (KP == kp && CP == cp) return b ? sweep_lds<bf16, kp, cp>() : sweep_lds<float, kp, cp>();
  GLA_LDS_CASE(64, 32) GLA_LDS_CASE(64, 64) GLA_LDS_CASE(128, 32) GLA_LDS_CASE(128, 64)
  GLA_LDS_CASE(256, 32) GLA_LDS_CASE(256, 64)
#undef GLA_LDS_CASE
  return 0;
}

template <typename T, int KP, int CP, bool REV, bool GB>
hipError_t launch_sweep_gb(const SweepArgs &a, hipStream_t st) {
  const size_t lds = GB ? SweepLayout<T, KP, CP>::total_gb : SweepLayout<T, KP, CP>::total;
  // once per instantiation (thread-safe static initialisation), at the maximum
  static const hipError_t attr = hipFuncSetAttribute((const void *)sweep_kernel<T, KP, CP, REV, GB>,
                                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  hipLaunchKernelGGL((sweep_kernel<T, KP, CP, REV, GB>), dim3(a.BH * a.ntiles), dim3(kThreads), lds, st, a);
  return hipGetLastError();
}

template <typename T, int KP, int CP, bool REV>
hipError_t launch_sweep_t(const SweepArgs &a, hipStream_t st) {
  if (a.LB) return launch_sweep_gb<T, KP, CP, REV, true>(a, st);
  return launch_sweep_gb<T, KP, CP, REV, false>(a, st);
}

template <typename T, bool REV>
hipError_t dispatch_sweep(const Shape &s, const SweepArgs &a, hipStream_t st) {
  const int KP = sweep_kp(s), CP = sweep_cp(s);
#define GLA_SWEEP_CASE(kp, cp) \
  if (KP == kp && CP == cp) return launch_sweep_t<T, kp, cp, REV>(a, st);
  GLA_SWEEP_CASE(64, 32) GLA_SWEEP_CASE(64, 64) GLA_SWEEP_CASE(128, 32) GLA_SWEEP_CASE(128, 64)
  if constexpr (sizeof(T) == 2) {
    GLA_SWEEP_CASE(256, 32) GLA_SWEEP_CASE(256, 64)
  }
#undef GLA_SWEEP_CASE
  return hipErrorInvalidValue;
}

SweepArgs sweep_args(const Shape &s) {
  SweepArgs a{};
  a.BH = s.BH; a.T = s.T; a.K = s.K; a.V = s.V; a.C = s.C; a.N = s.N;
  a.ntiles = (s.V + kTile - 1) / kTile;
  return a;
}

}  // namespace

size_t lds_fwd_main(const Shape &s) { return sweep_lds(s); }
size_t lds_bwd_dv(const Shape &s) { return sweep_lds(s); }

hipError_t launch_fwd_main(const Shape &s, const void *v, const void *lb, const float *S0, void *o, float *ST,
                           const Work &w, hipStream_t st) {
  SweepArgs a = sweep_args(s);
  a.X = w.Qt; a.Y = w.Kt; a.Z = v; a.P = w.P; a.gam = w.gam; a.R0 = S0; a.out = o; a.RN = ST; a.LB = lb;
  return s.io == IO_BF16 ? dispatch_sweep<bf16, false>(s, a, st) : dispatch_sweep<float, false>(s, a, st);
}

hipError_t launch_bwd_dv(const Shape &s, const void *dO, const void *lb, const float *dST, void *dv, float *dS0,
                         const Work &w, hipStream_t st) {
  SweepArgs a = sweep_args(s);
  a.X = w.Kt; a.Y = w.Qt; a.Z = dO; a.P = w.P; a.gam = w.gam; a.R0 = dST; a.out = dv; a.RN = dS0; a.LB = lb;
  return s.io == IO_BF16 ? dispatch_sweep<bf16, true>(s, a, st) : dispatch_sweep<float, true>(s, a, st);
}

}  // namespace gla
