// gla_ksweep.hip -- the two backward sweeps that tile the key features (App. B,
// Alg. 4/6 with the corrections listed in the header of gla_vsweep.hip, and the
// closed-form gate gradient of Sec. 4.3).
//
// Per chunk n (S_[n] = state before the chunk, dS_[n+1] = dL/dS after it, B =
// chunk-local inclusive cumsum of log alpha, Lambda = exp(B), Gamma =
// exp(B_last - B)):
//   dq_sweep (forward):  dq_inter = Lambda (.) (dO S_[n]^T)      (dq = dq_inter + dq_intra)
//                        S_[n+1] = Diag(gamma) S_[n] + (K (.) Gamma)^T V
//   dk_sweep (reverse):  dk_inter = Gamma (.) (V dS_[n+1]^T), dk = dk_inter + dk_intra
//                        dS_[n] = Diag(gamma) dS_[n+1] + (Q (.) Lambda)^T dO
//                        dlog alpha = revcumsum(q (.) dq - k (.) dk) + rowsum(S_T (.) dS_T)
// The intra-chunk terms (dq_intra, dk_intra and their share of the gate
// gradient) depend on no state; gla_intra.hip computes them chunk-parallel
// between the two sweeps: it adds dq_intra to the dq sweep's dq_inter and
// hands dk_intra and the gate-gradient share to the dk sweep.  Their one
// d_v-reducing input, dP = (dO V^T) (.) M, is formed here in the dq sweep,
// which streams V and dO through LDS anyway: for chunk n by the key tile
// n mod (number of key tiles) only, so each tile takes an equal share.
// dq, dk and the gate gradient reduce over d_v, so a workgroup owns 32 key
// features of one head for the whole sequence and holds the transposed state
// (value rows x 32 features, fp32) in matrix-core accumulators.
//
// Workgroup = 8 waves.  Value columns stream through LDS in slabs of 256
// (bf16; 128 for fp32); wave w holds the 32 x 32 state tile of value rows
// 32 w .. +32 of every slab as one 32x32 accumulator, so every operand fetched
// for the d_v-reducing products and the state update feeds a 32-wide output.
// Accumulator row m holds value 16 (m / 16) + 8 ((m / 4) % 2) + 4 ((m / 8) % 2)
// + m % 4 of the wave's 32, which makes the 8 values a lane holds for one
// 16-deep step contiguous: the tile is directly an operand of the next
// product, whose partner is one 16-byte LDS read; the update's transposed
// operand is read with LDS transpose reads pointed at the matching permuted
// columns.  Slab tiles are XOR-swizzled per row so that both read patterns are
// bank-conflict free.  The products that reduce over d_v leave one partial per
// state wave; these are pre-scaled and summed in two steps through LDS, then
// scaled per (row, feature) and added to the intra-chunk term.
// For bf16 the state operand and the gated update operand are split into bf16
// hi + lo, and dq_inter reaches the dk sweep in fp32, so that the gate
// gradient's long reverse sum keeps fp32 accuracy.
//
// NG (no gate and no gate gradient wanted: alpha = 1): every decay factor is
// 1 and the gated operands are k and q themselves, so the factor phase only
// stages k (q), the partials need no pre-scaling, the state needs no decay,
// and with no gate gradient to protect the state and update operands are
// used as single bf16 values (as the forward's inter-chunk products use them).
//
// General form (GB; App. C, a value-side gate beta as well): v and dO arrive
// as Vh = V (.) exp(-E) and Oh = dO (.) exp(E) (E the chunk-local cumsum of
// log beta, formed by gla_beta.hip), and the state's value rows decay by
// gb = exp(E_last) per chunk: S_[n+1] = (gamma S_[n] + (K (.) Gamma)^T Vh) gb
// in the dq sweep, D = dS_[n+1] gb before the dk sweep's products; the chunk's
// gb row is staged in LDS.
// For the value-side gate gradient the dq sweep also stores every chunk-end
// state S_[n+1] (io dtype, in the accumulators' own lane order), and the dk
// sweep, holding dS_[n+1] in the same order, forms this tile's
// colsum(S_[n+1] (.) dS_[n+1]): the exact carry of dlog beta into chunk n.
#include <type_traits>

#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

constexpr int kKT = 512;      // threads per workgroup
constexpr int kKF = 32;       // key features per workgroup
constexpr float kWide = 60.f;

typedef float f16v __attribute__((ext_vector_type(16)));

struct KsArgs {
  const void *q, *k, *la, *v, *dO;
  const void *dki, *dai;        // intra-chunk dk and in-chunk dA sums [BH][T][K] io (gla_intra.hip)
  const float *dat;             // [BH][N][K] chunk totals of the intra-chunk dA
  const float *S0, *dST;
  void *dk, *dla;
  float *dqr;                   // [BH][T][K] fp32 dq_inter: written by the dq sweep
  float *dP;                    // [BH][N][C][C] fp32 (dO V^T) (.) M per chunk, stored transposed ([s][t])
  float *cST;
  float *dla_part;  // scalar gate: [BH][KT][T] per-tile feature sums of the gate gradient
  const float *gbv; // general form: [BH][N][V] chunk decays exp(E_last) of the value-side gate
  void *Sb;         // general form: chunk-end states S_[n+1], accumulator-native layout (sb_index)
  float *cpart;     // general form: [BH][N][KT][V] per key tile colsum(S_[n+1] (.) dS_[n+1])
  int BH, T, K, V, C, N, KT;
  int sg;         // scalar gate: la is [BH][T], one value per step shared by every feature
  int ng;         // no gate and no gate gradient (la and dla NULL)
  float inv_tau;   // gate epilogue (0: la holds log alpha)
};

// Two slab buffers, so that the next slab is stored while the current one is
// multiplied; the per-(row, feature) gate values stay in registers.
template <typename T, int CP> struct KsLayout {
  static constexpr int VS = sizeof(T) == 2 ? 256 : 128;  // value columns per slab
  static constexpr int NWS = VS / 32;                     // waves holding state
  static constexpr int NP = NWS / 2;                      // partial slots are added in pairs (p, p + NP)
  static constexpr int LDV = VS;                          // slab rows are XOR-swizzled, not padded
  static constexpr int NB = CP / 16, NRG = CP / 4;
  // The gated update operand is stored feature-major ([32 features][rows]),
  // so a factor thread's four consecutive rows of one feature and a
  // fragment's eight consecutive rows are single 8/16-byte LDS accesses.
  static constexpr int LDTB = CP + (sizeof(T) == 2 ? 8 : 4);
  static constexpr int LDRG = NRG + 4;                        // row-group sums [32][NRG]
  static constexpr size_t slab = sizeof(T) * CP * LDV;
  // slab buffer b: the V tile at offV + 2 b slab, the dO tile after it
  static constexpr size_t offV = 0;
  static constexpr size_t offD = offV + slab;
  static constexpr size_t offBh = 4 * slab;                             // gated update operand (hi)
  static constexpr size_t offBl = offBh + sizeof(T) * kKF * LDTB;       // (lo, bf16 only)
  // per-wave partial sums [NWS][32 features][CP rows] fp32, 16-byte units
  // XOR-swizzled per row: aliased over the slab buffer of the chunk's last
  // slab, which is free from that slab's barrier until the next slab store
  // into it (two barriers later)
  static constexpr size_t offRed = offV;
  static_assert(4 * NWS * kKF * CP <= 2 * slab, "partials fit over a slab buffer");
  static constexpr size_t offOr = offBl + (sizeof(T) == 2 ? sizeof(T) * kKF * LDTB : 0);  // general form: gb row
  static constexpr size_t offRg = offOr + 4 * 1024;                     // row-group totals
  static constexpr size_t offSc = offRg + 4 * kKF * LDRG;               // per-block scale [NB][32]
  static constexpr size_t offG = offSc + 4 * NB * kKF;                  // gamma [32]
  static constexpr size_t offCar = offG + 4 * kKF;                      // carry [2][32]
  static constexpr size_t offRedS = offCar + 4 * 2 * kKF;               // final-state sums [8][32]
  static constexpr size_t offGrp = offRedS + 4 * 8 * kKF;               // dk: row-group sums of dA
  static constexpr size_t total = offGrp + 4 * kKF * LDRG;
};

// ------------------------------------------------------------- 32x32 tiles
// v_mfma_f32_32x32x16_bf16 (or 8 x v_mfma_f32_32x32x2f32): lane l = 32 g + j
// holds A[j][8g + i], B[8g + i][j] and D[8b + 4g + r][j] = acc[4b + r].
template <typename T> struct Mma32;
template <> struct Mma32<bf16> {
  static __device__ __forceinline__ f16v mma(f16v c, bf16x8 a, bf16x8 b) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma32<float> {
  static __device__ __forceinline__ f16v mma(f16v c, f8 a, f8 b) {
#pragma unroll
    for (int i = 0; i < 8; ++i) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[i], c, 0, 0, 0);
    return c;
  }
};
template <typename T> __device__ __forceinline__ f16v mma32(f16v c, frag_t<T> a, frag_t<T> b) {
  return Mma32<T>::mma(c, a, b);
}

// Value offset (within a wave's 32) of accumulator row m.
__device__ __forceinline__ int perm32(int m) {
  return 16 * (m >> 4) + 8 * ((m >> 2) & 1) + 4 * ((m >> 3) & 1) + (m & 3);
}
// Value offset of accumulator element e of lane group g.
__device__ __forceinline__ int acc_value(int e, int g) { return perm32(8 * (e >> 2) + 4 * g + (e & 3)); }

// Slab tiles: rows of kRowB bytes (256 bf16 or 128 fp32 values) whose 16-byte
// chunk c is stored at chunk c ^ swz(row).  The swizzle permutes the low four
// chunk bits only and the row offset starts at bit 9, so the byte offset of
// (row r0 + rr, chunk c0 / E + cc), with r0 a multiple of 16 and c0 a multiple
// of 16 values above the lane's own chunk bits cc, splits into a per-lane part
// XOR a wave-uniform column part, plus r0 kRowB: each lane keeps one base per
// read pattern and every read is one XOR (or none) away from it.
constexpr int kRowB = 512;
__device__ __forceinline__ int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

// Lane base of a row fragment (rows r0 + j, columns c0 + 8g; for fp32 half h
// holds columns + 4h).
template <typename T> __device__ __forceinline__ int row_lane_base(int h) {
  const int l = lane_id(), j = l & 31, g = l >> 5;
  const int ch = sizeof(T) == 2 ? g : 2 * g + h;
  return j * kRowB + ((ch ^ swz(j)) << 4);
}

// Row fragment from a slab: lane (g, j) gets X[r0 + j][c0 + 8g + i].
template <typename T>
__device__ __forceinline__ frag_t<T> ld_slab_row(const T *X, int lb0, int lb1, int r0, int c0) {
  const char *p = (const char *)X + r0 * kRowB;
  const int x = c0 * (int)sizeof(T);
  if constexpr (sizeof(T) == 2) {
    return *(const bf16x8 *)(p + (lb0 ^ x));
  } else {
    const f4 a = *(const f4 *)(p + (lb0 ^ x)), b = *(const f4 *)(p + (lb1 ^ x));
    return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
}

// Column fragment with permuted columns from a slab: lane (g, j) gets
// X[r0 + 8g + i][c0 + perm32(j)], c0 a multiple of 32.  For bf16 each LDS
// transpose read returns, to lane L of a 16-lane block, element L % 4 of the
// 4-vector loaded by lane 4 m + L / 4 (m = 0..3), so lane 4a + b of block
// (g, jh) points at row r0 + 8g + a (+4 for the second read) and columns
// c0 + 16 jh + 8 (b % 2) + 4 (b / 2) + 0..3; tr_lane_base(0 / 4) are the two
// lane bases.
__device__ __forceinline__ int tr_lane_base(int x4) {
  const int l = lane_id(), L = l & 15, jh = (l >> 4) & 1, g = l >> 5;
  const int row = 8 * g + (L >> 2) + x4;
  const int ch = 2 * jh + (L & 1);
  return row * kRowB + ((ch ^ swz(row)) << 4) + 8 * ((L >> 1) & 1);
}
template <typename T>
__device__ __forceinline__ frag_t<T> ld_slab_col_perm(const T *X, int lt0, int lt1, int r0, int c0) {
  if constexpr (sizeof(T) == 2) {
    const char *p = (const char *)X + r0 * kRowB;
    const int x = c0 * 2;
    s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p + (lt0 ^ x)));
    s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p + (lt1 ^ x)));
    s8 r = s8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, r);
  } else {
    const int l = lane_id(), g = l >> 5, col = c0 + perm32(l & 31);
    f8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = r0 + 8 * g + i;
      r[i] = X[row * (kRowB / 4) + (((col >> 2) ^ swz(row)) << 2) + (col & 3)];
    }
    return r;
  }
}

// Plain (unswizzled) row fragment: lane (g, j) gets X[r0 + j][c0 + 8g + i].
template <typename T>
__device__ __forceinline__ frag_t<T> ld_row32(const T *X, int ld, int r0, int c0) {
  const int l = lane_id();
  const T *p = X + (r0 + (l & 31)) * ld + c0 + 8 * (l >> 5);
  if constexpr (sizeof(T) == 2) {
    return *(const bf16x8 *)p;
  } else {
    const f4 a = *(const f4 *)p, b = *(const f4 *)(p + 4);
    return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
}

// The 8 accumulator values of 16-deep step st as an operand, split into bf16
// hi + lo (to ~16 mantissa bits; lo unused for fp32).
template <typename T>
__device__ __forceinline__ void acc_split32(const f16v &acc, int st, frag_t<T> &hi, frag_t<T> &lo) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    hi[i] = cvt<T>(acc[8 * st + i]);
    if constexpr (sizeof(T) == 2) lo[i] = cvt<T>(acc[8 * st + i] - (float)hi[i]);
  }
}

// ------------------------------------------------------------- 16x16 tiles
// Four consecutive elements as one 8-byte (bf16) or 16-byte (fp32) LDS store.
template <typename T> __device__ __forceinline__ void store4(T *p, const T (&v)[4]) {
  if constexpr (sizeof(T) == 2) *(bf16x4 *)p = bf16x4{v[0], v[1], v[2], v[3]};
  else *(f4 *)p = f4{v[0], v[1], v[2], v[3]};
}

// fp32 fragment from an fp32 LDS tile: lane (g, j) gets X[r0 + j][c0 + 8g + i]
// (16x16 layout, g = l / 16).
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
template <typename T> __device__ __forceinline__ void st_elem(__amdgpu_buffer_rsrc_t rs, uint32_t off, T v) {
  if constexpr (sizeof(T) == 2)
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), rs, off, 0, 0);
  else
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, v), rs, off, 0, 0);
}

// Byte offset of the i-th of a thread's four gate elements: the element's own
// offset `eoff` (per-feature gate), or the row's single value (scalar gate)
// at `sbase` + i elements, sbase = the thread's first row, or out of range for
// masked threads.
template <typename T> __device__ __forceinline__ uint32_t gate_off(int sg, uint32_t eoff, uint32_t sbase, int i) {
  return sg ? sbase + (uint32_t)(i * (int)sizeof(T)) : eoff;
}

// tile *= f by value row: f holds one factor per value; the four entries
// 4b .. 4b+3 of a lane's accumulator are four consecutive values, so each
// group is one 16-byte LDS read.
__device__ __forceinline__ void scale_rows(f16v &t, const float *f, int g) {
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const f4 x = *(const f4 *)(f + acc_value(4 * b, g));
#pragma unroll
    for (int r = 0; r < 4; ++r) t[4 * b + r] *= x[r];
  }
}

// Element index of lane l's 16 accumulator entries of state tile (bh, chunk
// n, key tile kt, slab sl, wave w) in the chunk-end state buffer.
__device__ __forceinline__ int64_t sb_index(int bh, int n, int N, int kt, int KT, int sl, int NSL, int w, int NWS,
                                            int l) {
  return (((((int64_t)bh * N + n) * KT + kt) * NSL + sl) * NWS + w) * 1024 + (int64_t)l * 16;
}

template <typename T> struct Tile16 { u32x4 r[sizeof(T) * 16 / 16]; };

// (each 16-byte vector is built whole: assigning its lanes one by one inside
// an unrolled loop was compiled into copies of the first lane for fp32)
template <typename T> __device__ __forceinline__ void store_tile16(T *p, const f16v &t) {
  if constexpr (sizeof(T) == 2) {
    auto pk = [&](int i) {
      return (uint32_t)__builtin_bit_cast(unsigned short, cvt<bf16>(t[2 * i])) |
             ((uint32_t)__builtin_bit_cast(unsigned short, cvt<bf16>(t[2 * i + 1])) << 16);
    };
    ((u32x4 *)p)[0] = u32x4{pk(0), pk(1), pk(2), pk(3)};
    ((u32x4 *)p)[1] = u32x4{pk(4), pk(5), pk(6), pk(7)};
  } else {
#pragma unroll
    for (int b = 0; b < 4; ++b) ((f4 *)p)[b] = f4{t[4 * b], t[4 * b + 1], t[4 * b + 2], t[4 * b + 3]};
  }
}

template <typename T> __device__ __forceinline__ float tile16_elem(const Tile16<T> &x, int e) {
  const uint32_t w = x.r[sizeof(T) == 2 ? e / 8 : e / 4][sizeof(T) == 2 ? (e / 2) % 4 : e % 4];
  if constexpr (sizeof(T) == 2) return __builtin_bit_cast(float, (e & 1) ? (w & 0xFFFF0000u) : (w << 16));
  else return __builtin_bit_cast(float, w);
}

// Sum over the 32 lanes of each half wave (every lane gets its half's sum).
__device__ __forceinline__ float half_wave_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x4E, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x141, 0xF, 0xF, false));
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x140, 0xF, 0xF, false));
  return x + __shfl_xor(x, 16);
}

// ------------------------------------------------------------- gate factors
// Cumulative-sum bookkeeping of one factor thread (feature fk, rows 4 frg ..
// +3 of the chunk), from the chunk's row-group totals in LDS.
struct Factors {
  float Bloc[4];  // block-local inclusive cumsum of log alpha
  float pre;      // log decay of the blocks before this thread's block
  float tot;      // log decay of this thread's 16-row block
  float blast;    // log decay of the whole chunk
  float bs[4];    // log decay of each 16-row block
};

template <int NRG, int LDRG>
__device__ __forceinline__ Factors chunk_factors(const float *sRg, const float (&c)[4], int frg, int blk,
                                                 int fk) {
  // blk (the thread's 16-row block) is uniform across the wave; frg % 4 (its
  // row group inside the block) is not
  Factors f;
  float *bs = f.bs;
  bs[1] = bs[2] = bs[3] = 0.f;
#pragma unroll
  for (int b = 0; b < NRG / 4; ++b) {
    const f4 v = *(const f4 *)(sRg + fk * LDRG + 4 * b);
    bs[b] = (v[0] + v[1]) + (v[2] + v[3]);
  }
  const f4 in_blk = *(const f4 *)(sRg + fk * LDRG + 4 * blk);
  f.blast = 0.f;
  f.pre = 0.f;
#pragma unroll
  for (int b = 0; b < NRG / 4; ++b) {
    f.blast += bs[b];
    if (b < blk) f.pre += bs[b];
  }
  f.tot = (in_blk[0] + in_blk[1]) + (in_blk[2] + in_blk[3]);
  const int q = frg & 3;
  const float ex = q == 0 ? 0.f : (q == 1 ? in_blk[0] : (q == 2 ? in_blk[0] + in_blk[1] : in_blk[0] + in_blk[1] + in_blk[2]));
#pragma unroll
  for (int i = 0; i < 4; ++i) f.Bloc[i] = ex + c[i];
  return f;
}

// Per-chunk gate data the factor threads publish: the block-level scale of the
// inter partials and gamma.
__device__ __forceinline__ void publish_decays(float *sSc, float *sG, const Factors &f, float scale_log,
                                               int frg, int fk, bool fv) {
  if ((frg & 3) == 0) sSc[(frg >> 2) * kKF + fk] = __expf(scale_log);
  if (frg == 0) sG[fk] = fv ? __expf(f.blast) : 0.f;
}

// Reduction of the d_v-reducing partials (rows t, feature j; 32-row tiles th):
// pre-scaled by the per-(16-row block, feature) factor, every state wave
// stores its tiles to its own slot; after one barrier the combine threads add
// the slots, pairwise (w, w + NP) in the order p = 0 .. NP-1.  Unit u (four
// rows) of feature row j sits at unit u ^ (j mod CP/4).
template <typename L, bool SCALE = true>
__device__ __forceinline__ void partials_store(f16v (&acc)[2], const float *sSc, float *sRed, int w, int g,
                                               int j) {
  constexpr int NTT = L::NB / 2, CP = L::NB * 16, UM = CP / 4 - 1;
  if constexpr (SCALE) {
    float sc[L::NB];
#pragma unroll
    for (int J = 0; J < L::NB; ++J) sc[J] = sSc[J * kKF + j];
#pragma unroll
    for (int th = 0; th < NTT; ++th)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[th][4 * b + r] *= sc[2 * th + (b >> 1)];
  }
  if (w < L::NWS) {
#pragma unroll
    for (int th = 0; th < NTT; ++th)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int u = 8 * th + 2 * b + g;
        *(f4 *)(sRed + (w * kKF + j) * CP + 4 * (u ^ (j & UM))) =
            f4{acc[th][4 * b], acc[th][4 * b + 1], acc[th][4 * b + 2], acc[th][4 * b + 3]};
      }
  }
}
// The sum of the slots for rows 4 frg .. +3 of feature fk.
template <typename L> __device__ __forceinline__ f4 partials_sum(const float *sRed, int fk, int frg) {
  constexpr int CP = L::NB * 16, UM = CP / 4 - 1;
  const int off = fk * CP + 4 * (frg ^ (fk & UM));
  auto slot = [&](int p) { return *(const f4 *)(sRed + p * kKF * CP + off); };
  f4 s = slot(0) + slot(L::NP);
#pragma unroll
  for (int p = 1; p < L::NP; ++p) s += slot(p) + slot(p + L::NP);
  return s;
}

// ============================================================== dq sweep
template <typename T, int CP, int NSL, bool PRE, bool GB, bool NG>
__global__ void __launch_bounds__(kKT) dq_sweep_kernel(KsArgs a) {
  using L = KsLayout<T, CP>;
  constexpr int VS = L::VS, NB = L::NB, NRG = L::NRG, NST = CP / 16, NTT = CP / 32;
  constexpr int NDT = CP == 64 ? 3 : 1;  // dP tiles on or below the diagonal, one per wave 0..NDT-1
  constexpr bool SPLIT = sizeof(T) == 2 && !NG;
  static_assert(VS * sizeof(T) == kRowB, "slab row size");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  // slab buffer b: V tile at b * 2 slab, dO tile right after it
  T *sV0 = (T *)(smem + L::offV), *sD0 = (T *)(smem + L::offD);
  T *sV1 = (T *)(smem + L::offV + 2 * L::slab), *sD1 = (T *)(smem + L::offD + 2 * L::slab);
  T *sBh = (T *)(smem + L::offBh), *sBl = (T *)(smem + L::offBl);
  float *sOr = (float *)(smem + L::offOr);
  float *sRg = (float *)(smem + L::offRg), *sSc = (float *)(smem + L::offSc);
  float *sG = (float *)(smem + L::offG);
  float *sRedS = (float *)(smem + L::offRedS);

  int bh, kt;
  xcd_map(a.BH, a.KT, bh, kt);
  const int tid = threadIdx.x, w = wave_id() & 7, l = lane_id();
  const int g = l >> 5, j = l & 31;  // 32x32 tile lane coordinates
  const bool sw = w < L::NWS;        // this wave holds state
  const int K = a.K, V = a.V, C = a.C, N = a.N, k0 = kt * kKF;
  const int fk = tid & 31, frg = tid >> 5;
  const bool fthr = frg < NRG;
  const int kf = k0 + fk;
  const bool fv = kf < K;
  const int esz = sizeof(T);
  const int lb0 = row_lane_base<T>(0), lb1 = row_lane_base<T>(1);
  const int lt0 = tr_lane_base(0), lt1 = tr_lane_base(4);

  f16v S[NSL];
#pragma unroll
  for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int vv = sl * VS + 32 * w + acc_value(e, g), kq = k0 + j;
      S[sl][e] = (a.S0 && sw && vv < V && kq < K) ? a.S0[((int64_t)bh * K + kq) * V + vv] : 0.f;
    }

  // ---- input streams
  const int lrow = a.sg ? 1 : K;  // gate elements per step
  const T *kh_ = (const T *)a.k + (int64_t)bh * a.T * K, *lah = (const T *)a.la + (int64_t)bh * a.T * lrow;
  const T *vh = (const T *)a.v + (int64_t)bh * a.T * V, *dOh = (const T *)a.dO + (int64_t)bh * a.T * V;
  uint32_t eoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * frg + i;
    eoff[i] = (fthr && row < C && fv) ? (uint32_t)((row * K + kf) * esz) : 0x80000000u;
  }
  // (C is a multiple of 4: a thread's four rows are all inside or all outside)
  const uint32_t sbase = (fthr && 4 * frg < C && fv) ? (uint32_t)(4 * frg * esz) : 0x80000000u;
  uint32_t fin_la[4], fin_k[4];
  // general form: the chunk's gb row (value v held by thread v mod 512)
  float gbr[2];
  auto fetch_gb = [&](int n) {
    const auto rs = make_rsrc(a.gbv + ((int64_t)bh * N + n) * V, (uint32_t)(V * 4));
#pragma unroll
    for (int i = 0; i < 2; ++i)
      gbr[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)((tid + kKT * i) * 4), 0, 0));
  };
  auto stage_gb = [&]() {  // into its 1024-float tile (d_v <= 1024)
#pragma unroll
    for (int i = 0; i < 2; ++i) sOr[tid + kKT * i] = gbr[i];
  };
  auto fetch_factors = [&](int n) {
    const int t0 = n * C;
    const uint32_t bytes = rsrc_bytes((int64_t)(a.T - t0) * K * esz);
    // an absent gate (alpha = 1) reads as log alpha = 0 from an empty range
    const auto rs_la = make_rsrc(a.la ? lah + (int64_t)t0 * lrow : kh_,
                                 a.la ? rsrc_bytes((int64_t)(a.T - t0) * lrow * esz) : 0u);
    const auto rs_k = make_rsrc(kh_ + (int64_t)t0 * K, bytes);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (!NG) fin_la[i] = ld_elem<T>(rs_la, gate_off<T>(a.sg, eoff[i], sbase, i));
      fin_k[i] = ld_elem<T>(rs_k, eoff[i]);
    }
    if constexpr (GB) fetch_gb(n);
  };
  TileLd<T, CP, VS, kKT> pv, pd;
  pv.init(V, C, VS);
  pd.init(V, C, VS);
  const int NQ = N * NSL;
  // part 0: the V slab, 1: the dO slab
  auto fetch_slab = [&](int q, int part) {
    q = min(q, NQ - 1);  // unconditional, see fetch_factors
    const int n = q / NSL, sl = q - n * NSL, t0 = n * C, c0 = sl * VS;
    const uint32_t bytes = rsrc_bytes(((int64_t)(a.T - t0) * V - c0) * esz);
    if (part == 0) pv.load(make_rsrc(vh + (int64_t)t0 * V + c0, bytes), V - c0);
    else pd.load(make_rsrc(dOh + (int64_t)t0 * V + c0, bytes), V - c0);
  };

  float *dqro = a.dqr + (int64_t)bh * a.T * K;
  float *dPg = a.dP + (int64_t)bh * N * C * C;
  // dP tiles: waves 0..NDT-1 each accumulate one whole 32x32 tile (t rows
  // 32 tr.., s columns 32 tc..: T00, T10, T11) over every slab of the chunks
  // this key tile forms dP for; wave NDT writes the zero tile above the diagonal
  const bool dpw = w < NDT;
  const int tr = (w == 1 || w == 2) ? 1 : 0, tc = w == 2 ? 1 : 0;
  const int pA = lb0 + 32 * tr * kRowB, pB = lb0 + 32 * tc * kRowB;
  const int pA1 = lb1 + 32 * tr * kRowB, pB1 = lb1 + 32 * tc * kRowB;

  // The gate factors of chunk n, in two parts around a barrier (the
  // row-group totals of log alpha are exchanged through LDS): part 1 forms the
  // cumsum of the thread's four rows from the prefetched gate rows, part 2
  // the gated keys K~ (hi/lo) in LDS, gamma and the block scales, and keeps
  // the block-local cumsum in registers for the chunk's combine.
  float c1[4], kv1[4];
  f4 bl4 = zero4();
  auto factors_part1 = [&](int n) {
    if constexpr (!NG) {
      const int rv = min(C, a.T - n * C);
      float x[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) x[i] = elem_f<T>(fin_la[i]);
      if constexpr (PRE) {  // gate epilogue
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = gate_la(x[i], a.inv_tau, fthr && fv && 4 * frg + i < rv);
      }
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s += x[i];
        c1[i] = s;
        kv1[i] = elem_f<T>(fin_k[i]);
      }
      if (fthr) sRg[fk * L::LDRG + frg] = s;
    }
  };
  auto factors_part2 = [&]() {
    if (fthr) {
      T hi4[4], lo4[4];
      if constexpr (NG) {
#pragma unroll
        for (int i = 0; i < 4; ++i) hi4[i] = cvt<T>(elem_f<T>(fin_k[i]));  // K~ = k
      } else {
        const Factors f = chunk_factors<NRG, L::LDRG>(sRg, c1, frg, w >> 1, fk);
        const float ekt = __expf(f.blast - f.pre - f.tot);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float kt_ = kv1[i] * __expf(f.tot - f.Bloc[i]) * ekt;
          hi4[i] = cvt<T>(kt_);
          lo4[i] = cvt<T>(kt_ - (float)hi4[i]);
          bl4[i] = f.Bloc[i];
        }
        publish_decays(sSc, sG, f, f.pre, frg, fk, fv);
      }
      store4<T>(sBh + fk * L::LDTB + 4 * frg, hi4);
      if constexpr (SPLIT) store4<T>(sBl + fk * L::LDTB + 4 * frg, lo4);
    }
    if constexpr (GB) stage_gb();
  };

  // Slabs are multiplied from one LDS buffer while the next slab, loaded one
  // step earlier, is stored into the other: one barrier per slab.  Prologue:
  // chunk 0's factors and slab 0 in LDS, slab 1 in flight.
  fetch_factors(0);
  fetch_slab(0, 0);
  fetch_slab(0, 1);
  factors_part1(0);
  pv.store_swz(sV0, L::LDV);
  pd.store_swz(sD0, L::LDV);
  fetch_slab(1, 0);
  fetch_slab(1, 1);
  __syncthreads();
  factors_part2();
  // unconditional (the last chunk re-reads itself) so that the wait counts
  // for the slab prefetches stay exact
  fetch_factors(min(1, N - 1));
  __syncthreads();

  for (int n = 0; n < N; ++n) {
    const int t0 = n * C;
    // ---- slabs: dq_inter partials (state before the chunk), update (and, for
    // one chunk in KT, the dP tiles)
    const bool mine = n % a.KT == kt;  // this key tile forms the chunk's dP
    f16v acc[2], accP;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[0][e] = acc[1][e] = accP[e] = 0.f;
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl) {
      const int q = n * NSL + sl;
      const bool b1 = (q & 1) != 0;  // this slab's buffer (even NSL: sl's parity)
      T *sV = b1 ? sV1 : sV0, *sD = b1 ? sD1 : sD0;    // this slab
      T *sVn = b1 ? sV0 : sV1, *sDn = b1 ? sD0 : sD1;  // the next one's buffer
      // the next slab (loaded during the previous step) into the other
      // buffer, which the previous step's barrier freed; no barrier before
      // this slab's products
      pv.store_swz(sVn, L::LDV);
      pd.store_swz(sDn, L::LDV);
      {
        if (sw) {
          // dq_inter += dO[:, this wave's 32 value rows] S^T
#pragma unroll
          for (int st = 0; st < 2; ++st) {
            frag_t<T> shi, slo;
            acc_split32<T>(S[sl], st, shi, slo);
#pragma unroll
            for (int th = 0; th < NTT; ++th) {
              const frag_t<T> ad = ld_slab_row<T>(sD, lb0, lb1, 32 * th, 32 * w + 16 * st);
              acc[th] = mma32<T>(acc[th], ad, shi);
              if constexpr (SPLIT) acc[th] = mma32<T>(acc[th], ad, slo);
            }
          }
          if constexpr (!NG) S[sl] *= sG[j];
        }
        // dP = dO V^T for this wave's tile (waves 0..NDT-1, chunks of this
        // key tile only), interleaved with the state update S^T <- gamma S^T
        // + V^T (K (.) Gamma) so that the two independent accumulation chains
        // hide each other's operand reads; the loads of the slab after the
        // next are issued in two halves between these products (pinned by
        // scheduling barriers) so that the memory pipeline drains meanwhile
        constexpr int NDS = VS / 16;    // dP steps per slab
        constexpr int UPD = NDS / NST;  // dP steps per update step
        auto slab_products = [&](auto with_dp) {
#pragma unroll
          for (int st = 0; st < NDS; ++st) {
            if constexpr (decltype(with_dp)::value)
              accP = mma32<T>(accP, ld_slab_row<T>(sD, pA, pA1, 0, 16 * st), ld_slab_row<T>(sV, pB, pB1, 0, 16 * st));
            if (st == 0 || st == NDS / 2) {
              __builtin_amdgcn_sched_barrier(0);
              fetch_slab(q + 2, st == 0 ? 0 : 1);
              __builtin_amdgcn_sched_barrier(0);
            }
            if (sw && (st + 1) % UPD == 0) {
              const int u = (st + 1) / UPD - 1;
              const frag_t<T> av = ld_slab_col_perm<T>(sV, lt0, lt1, 16 * u, 32 * w);
              S[sl] = mma32<T>(S[sl], av, ld_row32<T>(sBh, L::LDTB, 0, 16 * u));
              if constexpr (SPLIT) S[sl] = mma32<T>(S[sl], av, ld_row32<T>(sBl, L::LDTB, 0, 16 * u));
            }
          }
        };
        if (dpw && mine) slab_products(std::true_type{});
        else slab_products(std::false_type{});
        if constexpr (GB) {
          // S_[n+1] = (gamma S_[n] + K~^T Vh) gb, by value row
          static_assert(L::offOr % 16 == 0, "aligned factor rows");
          __builtin_amdgcn_sched_barrier(0);
          if (sw) {
            scale_rows(S[sl], sOr + sl * VS + 32 * w, g);
            store_tile16<T>((T *)a.Sb + sb_index(bh, n, N, kt, a.KT, sl, NSL, w, L::NWS, l), S[sl]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // (publishes the next slab; every read of this slab's buffer is done)
      __syncthreads();
    }

    // ---- dP of this key tile's chunks: masked, handed over transposed ([s][t])
    if (mine && (dpw || (CP == 64 && w == NDT))) {
      const bool zero_tile = !dpw;
      const int rt = zero_tile ? 0 : tr, ct = zero_tile ? 1 : tc;
      const int col = 32 * ct + j;
      const auto rs_dp = make_rsrc(dPg + (int64_t)n * C * C, (uint32_t)(C * C * 4));
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int t4 = 32 * rt + 8 * b + 4 * g;
        f4 v4;
#pragma unroll
        for (int r = 0; r < 4; ++r) v4[r] = (zero_tile || col > t4 + r) ? 0.f : accP[4 * b + r];
        const uint32_t off = (t4 < C && col < C) ? (uint32_t)((col * C + t4) * 4) : 0x80000000u;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v4), rs_dp, off, 0, 0);
      }
    }
    // ---- dq_inter partials, pre-scaled by exp(log decay before the block),
    // into the buffer of the chunk's last slab (the other one holds the next
    // chunk's first slab); the next chunk's factor part 1 alongside
    float *sRed = (float *)(smem + L::offRed + (((n * NSL + NSL - 1) & 1) ? 2 * L::slab : 0));
    partials_store<L, !NG>(acc, sSc, sRed, w, g, j);
    factors_part1(min(n + 1, N - 1));
    __syncthreads();

    // ---- dq_inter = Lambda (.) inter, per (row, feature)
    if (fthr) {
      const f4 in4 = partials_sum<L>(sRed, fk, frg);
      const auto rs_dqr = make_rsrc(dqro + (int64_t)t0 * K, rsrc_bytes((int64_t)(a.T - t0) * K * 4));
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float dqe = NG ? in4[i] : __expf(bl4[i]) * in4[i];
        // rows past the sequence end, past the chunk or of absent features
        // fall outside the buffer range and are dropped
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, dqe), rs_dqr,
                                              eoff[i] == 0x80000000u ? eoff[i] : eoff[i] / esz * 4, 0, 0);
      }
    }
    // ---- the next chunk's factor part 2 (the last chunk redoes its own);
    // the barrier publishes its tiles and orders the combine's reads of the
    // partials before the next slab store into their buffer
    factors_part2();
    fetch_factors(min(n + 2, N - 1));
    __syncthreads();
  }

  // ---- final-state term of the gate gradient: rowsum(S_T (.) dS_T) per feature
  if (!NG && a.dST) {
    float part = 0.f;
    if (sw) {
#pragma unroll
      for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int vv = sl * VS + 32 * w + acc_value(e, g), kq = k0 + j;
          if (vv < V && kq < K) part += S[sl][e] * a.dST[((int64_t)bh * K + kq) * V + vv];
        }
    }
    part += __shfl_xor(part, 32);
    if (g == 0) sRedS[w * kKF + j] = part;
    __syncthreads();
    if (tid < kKF && k0 + tid < K) {
      float s = 0.f;
#pragma unroll
      for (int w2 = 0; w2 < 8; ++w2) s += sRedS[w2 * kKF + tid];
      a.cST[(int64_t)bh * K + k0 + tid] = s;
    }
  }
}

// ============================================================== dk sweep
template <typename T, int CP, int NSL, bool PRE, bool GB, bool NG>
__global__ void __launch_bounds__(kKT) dk_sweep_kernel(KsArgs a) {
  using L = KsLayout<T, CP>;
  constexpr int VS = L::VS, NB = L::NB, NRG = L::NRG, NST = CP / 16, NTT = CP / 32;
  constexpr bool SPLIT = sizeof(T) == 2 && !NG;
  static_assert(VS * sizeof(T) == kRowB, "slab row size");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  // slab buffer b: V tile at b * 2 slab, dO tile right after it
  T *sV0 = (T *)(smem + L::offV), *sD0 = (T *)(smem + L::offD);
  T *sV1 = (T *)(smem + L::offV + 2 * L::slab), *sD1 = (T *)(smem + L::offD + 2 * L::slab);
  T *sBh = (T *)(smem + L::offBh), *sBl = (T *)(smem + L::offBl);
  float *sOr = (float *)(smem + L::offOr);
  float *sRg = (float *)(smem + L::offRg), *sSc = (float *)(smem + L::offSc);
  float *sG = (float *)(smem + L::offG);
  float *sCar = (float *)(smem + L::offCar);
  float *sGrp = (float *)(smem + L::offGrp);

  int bh, kt;
  xcd_map(a.BH, a.KT, bh, kt);
  const int tid = threadIdx.x, w = wave_id() & 7, l = lane_id();
  const int g = l >> 5, j = l & 31;
  const bool sw = w < L::NWS;
  const int K = a.K, V = a.V, C = a.C, N = a.N, k0 = kt * kKF;
  const int fk = tid & 31, frg = tid >> 5;
  const bool fthr = frg < NRG;
  const int kf = k0 + fk;
  const bool fv = kf < K;
  const int esz = sizeof(T);
  const int lb0 = row_lane_base<T>(0), lb1 = row_lane_base<T>(1);
  const int lt0 = tr_lane_base(0), lt1 = tr_lane_base(4);

  if (tid < kKF) sCar[tid] = (a.cST && k0 + tid < K) ? a.cST[(int64_t)bh * K + k0 + tid] : 0.f;

  f16v dS[NSL];
#pragma unroll
  for (int sl = 0; sl < NSL; ++sl)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int vv = sl * VS + 32 * w + acc_value(e, g), kq = k0 + j;
      dS[sl][e] = (a.dST && sw && vv < V && kq < K) ? a.dST[((int64_t)bh * K + kq) * V + vv] : 0.f;
    }

  const T *qh_ = (const T *)a.q + (int64_t)bh * a.T * K, *kh_ = (const T *)a.k + (int64_t)bh * a.T * K;
  const int lrow = a.sg ? 1 : K;  // gate elements per step
  const T *lah = (const T *)a.la + (int64_t)bh * a.T * lrow;
  const float *dqrh = a.dqr + (int64_t)bh * a.T * K;
  const T *dkih = (const T *)a.dki + (int64_t)bh * a.T * K, *daih = (const T *)a.dai + (int64_t)bh * a.T * K;
  const float *dath = a.dat + (int64_t)bh * N * K;
  const T *vh = (const T *)a.v + (int64_t)bh * a.T * V, *dOh = (const T *)a.dO + (int64_t)bh * a.T * V;
  uint32_t eoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * frg + i;
    eoff[i] = (fthr && row < C && fv) ? (uint32_t)((row * K + kf) * esz) : 0x80000000u;
  }
  // (C is a multiple of 4: a thread's four rows are all inside or all outside)
  const uint32_t sbase = (fthr && 4 * frg < C && fv) ? (uint32_t)(4 * frg * esz) : 0x80000000u;
  uint32_t fin_la[4], fin_q[4], fin_k[4], fin_dqr[4], fin_dki[4], fin_dai[4], fin_dat;
  // general form: the chunk's gb row (value v held by thread v mod 512)
  float gbr[2];
  auto fetch_gb = [&](int n) {
    const auto rs = make_rsrc(a.gbv + ((int64_t)bh * N + n) * V, (uint32_t)(V * 4));
#pragma unroll
    for (int i = 0; i < 2; ++i)
      gbr[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (uint32_t)((tid + kKT * i) * 4), 0, 0));
  };
  auto stage_gb = [&]() {  // into its 1024-float tile (d_v <= 1024)
#pragma unroll
    for (int i = 0; i < 2; ++i) sOr[tid + kKT * i] = gbr[i];
  };
  // general form: the dq sweep's chunk-end state tile, one slab ahead
  Tile16<T> svr;
  auto fetch_sv = [&](int n, int sl) {
    if (sw) {
      const u32x4 *p = (const u32x4 *)((const T *)a.Sb + sb_index(bh, n, N, kt, a.KT, sl, NSL, w, L::NWS, l));
#pragma unroll
      for (int i = 0; i < (int)(sizeof(svr.r) / 16); ++i) svr.r[i] = p[i];
    }
  };
  auto fetch_factors = [&](int n) {
    const int t0 = n * C;
    const uint32_t bytes = rsrc_bytes((int64_t)(a.T - t0) * K * esz);
    // an absent gate (alpha = 1) reads as log alpha = 0 from an empty range
    const auto rs_la = make_rsrc(a.la ? lah + (int64_t)t0 * lrow : kh_,
                                 a.la ? rsrc_bytes((int64_t)(a.T - t0) * lrow * esz) : 0u);
    const auto rs_q = make_rsrc(qh_ + (int64_t)t0 * K, bytes);
    const auto rs_k = make_rsrc(kh_ + (int64_t)t0 * K, bytes);
    const auto rs_dqr = make_rsrc(dqrh + (int64_t)t0 * K, rsrc_bytes((int64_t)(a.T - t0) * K * 4));
    const auto rs_dki = make_rsrc(dkih + (int64_t)t0 * K, bytes);
    const auto rs_dai = make_rsrc(daih + (int64_t)t0 * K, bytes);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fin_q[i] = ld_elem<T>(rs_q, eoff[i]);
      fin_dki[i] = ld_elem<T>(rs_dki, eoff[i]);
      if constexpr (!NG) {
        fin_la[i] = ld_elem<T>(rs_la, gate_off<T>(a.sg, eoff[i], sbase, i));
        fin_k[i] = ld_elem<T>(rs_k, eoff[i]);
        fin_dqr[i] = __builtin_amdgcn_raw_buffer_load_b32(rs_dqr, eoff[i] == 0x80000000u ? eoff[i] : eoff[i] / esz * 4, 0, 0);
        fin_dai[i] = ld_elem<T>(rs_dai, eoff[i]);
      }
    }
    if constexpr (!NG)
      fin_dat = __builtin_amdgcn_raw_buffer_load_b32(make_rsrc(dath + (int64_t)n * K, (uint32_t)(K * 4)),
                                                     fv ? (uint32_t)(kf * 4) : 0x80000000u, 0, 0);
    if constexpr (GB) fetch_gb(n);
  };
  TileLd<T, CP, VS, kKT> pv, pd;
  pv.init(V, C, VS);
  pd.init(V, C, VS);
  const int NQ = N * NSL;
  auto fetch_slab = [&](int q, int part) {  // as in the dq sweep
    q = min(q, NQ - 1);
    const int n = N - 1 - q / NSL, sl = q % NSL, t0 = n * C, c0 = sl * VS;
    const uint32_t bytes = rsrc_bytes(((int64_t)(a.T - t0) * V - c0) * esz);
    if (part == 0) pv.load(make_rsrc(vh + (int64_t)t0 * V + c0, bytes), V - c0);
    else pd.load(make_rsrc(dOh + (int64_t)t0 * V + c0, bytes), V - c0);
  };

  T *dko = (T *)a.dk + (int64_t)bh * a.T * K, *dlao = (T *)a.dla + (int64_t)bh * a.T * K;

  // Per-(row, feature) values of a chunk, kept in registers from its factor
  // phase to its combine (cur: the chunk being swept, nxt: the next one in
  // the sweep, formed at the boundary before it): the gate argument zc (for
  // the gate gradient), the block-local cumsum, the block total, k, q dq_inter,
  // and the intra kernel's dk_intra, dA_intra share and chunk total.
  struct ChunkVals {
    float c[4], kv[4], qdq[4], zc[4], dki[4], dai[4], dat, tot;
  };
  ChunkVals cur, nxt;
  // factor part 1 of chunk n: its values from the prefetched rows, and the
  // row-group totals of log alpha into LDS
  auto factors_part1 = [&](int n) {
    const int rv = min(C, a.T - n * C);
#pragma unroll
    for (int i = 0; i < 4; ++i) nxt.dki[i] = elem_f<T>(fin_dki[i]);
    if constexpr (!NG) {
      nxt.dat = __builtin_bit_cast(float, fin_dat);
      float x[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[i] = nxt.zc[i] = elem_f<T>(fin_la[i]);
        nxt.dai[i] = elem_f<T>(fin_dai[i]);
      }
      if constexpr (PRE) {  // gate epilogue
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = gate_la(x[i], a.inv_tau, fthr && fv && 4 * frg + i < rv);
      }
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s += x[i];
        nxt.c[i] = s;
        nxt.kv[i] = elem_f<T>(fin_k[i]);
        nxt.qdq[i] = elem_f<T>(fin_q[i]) * __builtin_bit_cast(float, fin_dqr[i]);
      }
      if (fthr) sRg[fk * L::LDRG + frg] = s;
    }
  };
  // factor part 2: Q~ (hi/lo) into LDS, gamma and the block scales; the
  // block-local cumsum replaces the chunk's cumsum in nxt.c
  auto factors_part2 = [&]() {
    if (fthr) {
      T hi4[4], lo4[4];
      if constexpr (NG) {
#pragma unroll
        for (int i = 0; i < 4; ++i) hi4[i] = cvt<T>(elem_f<T>(fin_q[i]));  // Q~ = q
      } else {
        const Factors f = chunk_factors<NRG, L::LDRG>(sRg, nxt.c, frg, w >> 1, fk);
        nxt.tot = f.tot;
        const float epre = __expf(f.pre);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float qt = elem_f<T>(fin_q[i]) * __expf(f.Bloc[i]) * epre;
          hi4[i] = cvt<T>(qt);
          lo4[i] = cvt<T>(qt - (float)hi4[i]);
          nxt.c[i] = f.Bloc[i];
        }
        publish_decays(sSc, sG, f, f.blast - f.pre - f.tot, frg, fk, fv);
      }
      store4<T>(sBh + fk * L::LDTB + 4 * frg, hi4);
      if constexpr (SPLIT) store4<T>(sBl + fk * L::LDTB + 4 * frg, lo4);
    }
    if constexpr (GB) stage_gb();
  };

  // Slabs are multiplied from one LDS buffer while the next is stored into the
  // other (as in the dq sweep).  Prologue: the last chunk's factors and its
  // first slab in LDS, the second in flight.
  fetch_factors(N - 1);
  fetch_slab(0, 0);
  fetch_slab(0, 1);
  factors_part1(N - 1);
  pv.store_swz(sV0, L::LDV);
  pd.store_swz(sD0, L::LDV);
  fetch_slab(1, 0);
  fetch_slab(1, 1);
  __syncthreads();
  factors_part2();
  fetch_factors(max(N - 2, 0));  // unconditional, see the dq sweep
  cur = nxt;
  if constexpr (GB) fetch_sv(N - 1, 0);
  __syncthreads();

  for (int it = 0; it < N; ++it) {
    const int n = N - 1 - it;
    const int t0 = n * C;

    // ---- slabs: dk_inter partials (dS after the chunk), then the dS update
    f16v acc[2];
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[0][e] = acc[1][e] = 0.f;
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl) {
      const int q = it * NSL + sl;
      const bool b1 = (q & 1) != 0;  // this slab's buffer
      T *sV = b1 ? sV1 : sV0, *sD = b1 ? sD1 : sD0;
      // the next slab into the other buffer (freed by the previous barrier)
      pv.store_swz(b1 ? sV0 : sV1, L::LDV);
      pd.store_swz(b1 ? sD0 : sD1, L::LDV);
      if constexpr (GB) {
        // this tile's colsum(S_[n+1] (.) dS_[n+1]) per value: the carry of the
        // value-side gate gradient into chunk n
        float *cp = a.cpart + (((int64_t)bh * N + n) * a.KT + kt) * V;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float cs = half_wave_sum(sw ? dS[sl][e] * tile16_elem<T>(svr, e) : 0.f);
          const int vv = sl * VS + 32 * w + acc_value(e, g);
          if (sw && j == 0 && vv < V) cp[vv] = cs;
        }
        if (sl + 1 < NSL) fetch_sv(n, sl + 1);
        // D = dS_[n+1] gb, by value row, before the chunk's products
        __builtin_amdgcn_sched_barrier(0);
        if (sw) scale_rows(dS[sl], sOr + sl * VS + 32 * w, g);
        __builtin_amdgcn_sched_barrier(0);
      }
      // the loads of the slab after the next go out in two halves between
      // the dk_inter products (every wave, so that each issues its share)
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        if (sw) {
          // dk_inter += V[:, this wave's 32 value rows] dS^T
          frag_t<T> shi, slo;
          acc_split32<T>(dS[sl], st, shi, slo);
#pragma unroll
          for (int th = 0; th < NTT; ++th) {
            const frag_t<T> av = ld_slab_row<T>(sV, lb0, lb1, 32 * th, 32 * w + 16 * st);
            acc[th] = mma32<T>(acc[th], av, shi);
            if constexpr (SPLIT) acc[th] = mma32<T>(acc[th], av, slo);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        fetch_slab(q + 2, st);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (sw) {
        // dS^T <- gamma dS^T + dO^T (Q (.) Lambda)
        if constexpr (!NG) dS[sl] *= sG[j];
#pragma unroll
        for (int st = 0; st < NST; ++st) {
          const frag_t<T> ad = ld_slab_col_perm<T>(sD, lt0, lt1, 16 * st, 32 * w);
          dS[sl] = mma32<T>(dS[sl], ad, ld_row32<T>(sBh, L::LDTB, 0, 16 * st));
          if constexpr (SPLIT) dS[sl] = mma32<T>(dS[sl], ad, ld_row32<T>(sBl, L::LDTB, 0, 16 * st));
        }
      }
      // (publishes the next slab; every read of this slab's buffer is done)
      __syncthreads();
    }

    // the next chunk's first state tile, in flight during the combine phases
    if constexpr (GB) fetch_sv(max(n - 1, 0), 0);
    // ---- dk_inter partials, pre-scaled by exp(B_last - B at the block's end),
    // into the buffer of the chunk's last slab
    float *sRed = (float *)(smem + L::offRed + (((it * NSL + NSL - 1) & 1) ? 2 * L::slab : 0));
    partials_store<L, !NG>(acc, sSc, sRed, w, g, j);
    __syncthreads();

    if constexpr (NG) {
      // dk = dk_inter + dk_intra; the next chunk's factors
      if (fthr) {
        const f4 in4 = partials_sum<L>(sRed, fk, frg);
        const auto rs_dk = make_rsrc(dko + (int64_t)t0 * K, rsrc_bytes((int64_t)(a.T - t0) * K * esz));
#pragma unroll
        for (int i = 0; i < 4; ++i) st_elem<T>(rs_dk, eoff[i], cvt<T>(in4[i] + cur.dki[i]));
      }
      factors_part1(max(n - 1, 0));
      factors_part2();
      fetch_factors(max(n - 2, 0));
      cur = nxt;
      // (publishes Q~; orders the reads of the partials before the next
      // slab store into their buffer)
      __syncthreads();
      continue;
    }

    // ---- dk_inter = Gamma (.) inter; dk = dk_inter + dk_intra; dA = q dq - k dk
    // (inter parts here; the intra parts arrive summed) and in-chunk reverse
    // sums; the next chunk's factor part 1 alongside
    float dA[4];
    if (fthr) {
      const f4 in4 = partials_sum<L>(sRed, fk, frg);
      const auto rs_dk = make_rsrc(dko + (int64_t)t0 * K, rsrc_bytes((int64_t)(a.T - t0) * K * esz));
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float dke = __expf(cur.tot - cur.c[i]) * in4[i];
        dA[i] = cur.qdq[i] - cur.kv[i] * dke;
        st_elem<T>(rs_dk, eoff[i], cvt<T>(dke + cur.dki[i]));
      }
      float s = 0.f;
#pragma unroll
      for (int i = 3; i >= 0; --i) {
        s += dA[i];
        dA[i] = s;
      }
      sGrp[fk * L::LDRG + frg] = s;
    }
    factors_part1(max(n - 1, 0));
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
      for (int i = 0; i < 4; ++i) dA[i] += later + cur.dai[i];
      if (a.sg) {
        // scalar gate: this tile's sum over its features, per row (rows past
        // the sequence end fall outside the range); the key tiles are added,
        // and the gate epilogue's chain rule applied, by sgate_dla_kernel
        if (a.dla) {
          float rr[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) rr[i] = half_wave_sum(fv ? dA[i] : 0.f);
          if (fk == 0) {
            const auto rs_p = make_rsrc(a.dla_part + ((int64_t)bh * a.KT + kt) * a.T + t0,
                                        rsrc_bytes((int64_t)(a.T - t0) * 4));
#pragma unroll
            for (int i = 0; i < 4; ++i)
              __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, rr[i]), rs_p,
                                                    (uint32_t)((4 * frg + i) * 4), 0, 0);
          }
        }
      } else {
        // an absent gate gradient is dropped through an empty range
        const auto rs_dla = make_rsrc(a.dla ? dlao + (int64_t)t0 * K : dko,
                                      a.dla ? rsrc_bytes((int64_t)(a.T - t0) * K * esz) : 0u);
        if constexpr (PRE) {  // gate epilogue: dL/dz = dL/dlog alpha * sigmoid(-z) / tau
#pragma unroll
          for (int i = 0; i < 4; ++i) dA[i] *= gate_dla_dg(cur.zc[i], a.inv_tau);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) st_elem<T>(rs_dla, eoff[i], cvt<T>(dA[i]));
      }
      if (frg == 0) sCar[((it + 1) & 1) * kKF + fk] = all + cur.dat;
    }
    // ---- the next chunk's factor part 2 (the last chunk redoes its own); the
    // barrier publishes its tiles before the next chunk's products
    factors_part2();
    fetch_factors(max(n - 2, 0));
    cur = nxt;
    __syncthreads();
  }
}

// Scalar gate: dlog gamma[bh][t] = sum over the key tiles of the per-tile
// feature sums, in tile order; with the gate epilogue, times
// sigmoid(-z) / tau of the scalar pre-activation z.
template <typename T>
__global__ void __launch_bounds__(256) sgate_dla_kernel(const float *part, const void *z, void *dla, int64_t n,
                                                        int steps, int KT, float inv_tau) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const int64_t bh = i / steps, t = i - bh * steps;
    const float *p = part + bh * KT * steps + t;
    float s = 0.f;
    for (int kt = 0; kt < KT; ++kt) s += p[(int64_t)kt * steps];
    if (inv_tau != 0.f) s *= gate_dla_dg((float)((const T *)z)[i], inv_tau);
    ((T *)dla)[i] = cvt<T>(s);
  }
}

// ============================================================== launchers
int ks_cp(const Shape &s) { return s.C <= 32 ? 32 : 64; }
int ks_nsl(const Shape &s) {
  const int vs = s.io == IO_BF16 ? 256 : 128;
  const int n = (s.V + vs - 1) / vs;
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
  a.inv_tau = s.inv_tau;
  a.sg = s.sgate ? 1 : 0;
  a.KT = (s.K + kKF - 1) / kKF;
  return a;
}

template <bool DQ, typename T, int CP, int NSL, bool PRE, bool GB, bool NG>
hipError_t launch_ks_pre(const KsArgs &a, hipStream_t st) {
  const size_t lds = KsLayout<T, CP>::total;
  // once per instantiation (thread-safe static initialisation), at the maximum
  static const hipError_t attr =
      hipFuncSetAttribute(DQ ? (const void *)dq_sweep_kernel<T, CP, NSL, PRE, GB, NG>
                             : (const void *)dk_sweep_kernel<T, CP, NSL, PRE, GB, NG>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
  (void)attr;
  if constexpr (DQ)
    hipLaunchKernelGGL((dq_sweep_kernel<T, CP, NSL, PRE, GB, NG>), dim3(a.BH * a.KT), dim3(kKT), lds, st, a);
  else
    hipLaunchKernelGGL((dk_sweep_kernel<T, CP, NSL, PRE, GB, NG>), dim3(a.BH * a.KT), dim3(kKT), lds, st, a);
  return hipGetLastError();
}

// PRE: the gate argument is the pre-activation of the gate epilogue.  GB: the
// general form (value-side gate; the entry point rules out PRE with it).  NG:
// no gate and no gate gradient (never with GB).
template <bool DQ, typename T, int CP, int NSL>
hipError_t launch_ks_t(const KsArgs &a, hipStream_t st) {
  if (a.gbv) return launch_ks_pre<DQ, T, CP, NSL, false, true, false>(a, st);
  if (a.ng) return launch_ks_pre<DQ, T, CP, NSL, false, false, true>(a, st);
  return a.inv_tau != 0.f ? launch_ks_pre<DQ, T, CP, NSL, true, false, false>(a, st)
                          : launch_ks_pre<DQ, T, CP, NSL, false, false, false>(a, st);
}

template <bool DQ, typename T, int CP>
hipError_t dispatch_ks_cp(const Shape &s, const KsArgs &a, hipStream_t st) {
  switch (ks_nsl(s)) {
    case 1: return launch_ks_t<DQ, T, CP, 1>(a, st);
    case 2: return launch_ks_t<DQ, T, CP, 2>(a, st);
    case 4: return launch_ks_t<DQ, T, CP, 4>(a, st);
    default:
      // eight slabs only arise for fp32 (d_v <= 1024 is four 256-wide bf16 slabs)
      if constexpr (sizeof(T) == 4) return launch_ks_t<DQ, T, CP, 8>(a, st);
      return hipErrorInvalidValue;
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

size_t ks_state_bytes(const Shape &s) {
  const int vs = s.io == IO_BF16 ? 256 : 128;
  const int64_t kt = (s.K + kKF - 1) / kKF;
  return (size_t)s.BH * s.N * kt * ks_nsl(s) * vs * kKF * s.esz();
}
size_t lds_bwd_dk(const Shape &s) { return ks_lds(s); }

hipError_t launch_bwd_dq(const Shape &s, const void *k, const void *la, const void *v,
                         const float *S0, const void *dO, const float *dST,
                         const Work &w, hipStream_t st, bool ng, bool gb_on) {
  KsArgs a = ks_args(s);
  a.k = k; a.la = la; a.v = v; a.dO = dO; a.S0 = S0; a.dST = dST; a.dqr = w.dqr;
  a.dP = w.dP; a.cST = w.cST;
  a.ng = ng && !gb_on;
  if (gb_on) { a.gbv = w.gb; a.Sb = w.Sb; }
  return dispatch_ks<true>(s, a, st);
}

hipError_t launch_bwd_dk(const Shape &s, const void *q, const void *k, const void *la,
                         const void *v, const void *dO, const float *dST, const void *dq,
                         void *dk, void *dla, const Work &w, hipStream_t st, bool gb_on) {
  KsArgs a = ks_args(s);
  if (gb_on) { a.gbv = w.gb; a.Sb = w.Sb; a.cpart = w.cpart; }
  a.q = q; a.k = k; a.la = la; a.v = v; a.dO = dO; a.dST = dST; a.dqr = w.dqr;
  a.dki = w.dki; a.dai = w.dai; a.dat = w.dat;
  a.dk = dk; a.dla = dla; a.cST = dST ? w.cST : nullptr; a.dla_part = w.dla_part;
  a.ng = !la && !dla && !gb_on;
  hipError_t e = dispatch_ks<false>(s, a, st);
  if (e != hipSuccess || !s.sgate || !dla) return e;
  const int64_t n = (int64_t)s.BH * s.T;
  const int blocks = (int)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192);
  if (s.io == IO_BF16)
    hipLaunchKernelGGL(sgate_dla_kernel<bf16>, dim3(blocks), dim3(256), 0, st, w.dla_part, la, dla, n, s.T, a.KT,
                       s.inv_tau);
  else
    hipLaunchKernelGGL(sgate_dla_kernel<float>, dim3(blocks), dim3(256), 0, st, w.dla_part, la, dla, n, s.T, a.KT,
                       s.inv_tau);
  return hipGetLastError();
}

}  // namespace gla
