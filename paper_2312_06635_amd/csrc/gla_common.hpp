// gla_common.hpp -- device building blocks shared by the GLA kernels (gfx950).
//
// Matrix-core tiles are 16x16 outputs with a 32-deep reduction per step:
//   bf16 : one v_mfma_f32_16x16x32_bf16
//   fp32 : eight v_mfma_f32_16x16x4_f32 (so the fp32 path never rounds to bf16)
// A "fragment" is the 8 reduction-slot values one lane contributes.  For lane
// l = 16 g + j (g = l / 16 in 0..3, j = l % 16):
//   A operand : row j of the 16-row tile, reduction slots 8g .. 8g+7
//   B operand : column j of the tile,    reduction slots 8g .. 8g+7
//   D (acc)   : column j, rows 4g .. 4g+3 (4 fp32 per lane)
// Any slot-to-index mapping is valid as long as A and B agree; a 16x16
// accumulator pair provides slots 0..3 and 4..7 from rows 4g..4g+3 of each
// accumulator (see acc_frag), which the kernels match by permuting the order
// in which the state's key features are laid out.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gla {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef short s8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s4 lds_s4;

template <typename T> struct Mma;

template <> struct Mma<bf16> {
  using frag = bf16x8;
  static __device__ __forceinline__ f4 mma(f4 c, frag a, frag b) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  using frag = f8;
  static __device__ __forceinline__ f4 mma(f4 c, frag a, frag b) {
#pragma unroll
    for (int i = 0; i < 8; ++i) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[i], c, 0, 0, 0);
    return c;
  }
};

template <typename T> using frag_t = typename Mma<T>::frag;

template <typename T> __device__ __forceinline__ f4 mma(f4 c, frag_t<T> a, frag_t<T> b) {
  return Mma<T>::mma(c, a, b);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
// The wave index is uniform across a wave; reading it through readfirstlane
// lets the compiler keep it (and every branch on it) in scalar registers.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

template <typename T> __device__ __forceinline__ T cvt(float x);
template <> __device__ __forceinline__ float cvt<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 cvt<bf16>(float x) { return (bf16)x; }

__device__ __forceinline__ f4 zero4() { return f4{0.f, 0.f, 0.f, 0.f}; }

constexpr float kLog2e = 1.4426950408889634f;
// 2^x by the hardware exponential (v_exp_f32): exponents held in units of
// log2 save the multiply by log2(e) that an exp() would add.
__device__ __forceinline__ float exp2f_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// log alpha from the gate argument g: g itself when inv_tau == 0, else the
// GLA gate epilogue alpha = sigmoid(g)^(1/tau) of Sec. 4.4, i.e. log alpha =
// logsigmoid(g) / tau with logsigmoid(g) = min(g, 0) - log1p(e), e =
// exp(-|g|) in (0, 1]: log1p(e) is log(1 + e), or e (1 - e / 2) below 1e-3,
// where 1 + e would lose e's low bits (absolute error < 1e-9 either way).
// Elements outside the sequence (ok == false) contribute log alpha = 0.
__device__ __forceinline__ float gate_la(float g, float inv_tau, bool ok) {
  if (inv_tau == 0.f) return g;
  const float e = __expf(-fabsf(g));
  const float l1p = e < 1e-3f ? e * (1.f - 0.5f * e) : __logf(1.f + e);
  return ok ? (fminf(g, 0.f) - l1p) * inv_tau : 0.f;
}
// d log alpha / d g: 1, or sigmoid(-g) / tau for the gate epilogue.
__device__ __forceinline__ float gate_dla_dg(float g, float inv_tau) {
  return inv_tau == 0.f ? 1.f : inv_tau / (1.f + __expf(g));
}

// ---------------------------------------------------------------- fragments
// All loaders read LDS tiles stored row-major with leading dimension `ld`
// (in elements).

// A/B fragment whose reduction index runs along a row:
// lane (g, j) gets X[r0 + j][c0 + 8g + i], i = 0..7.
template <typename T>
__device__ __forceinline__ frag_t<T> ld_row(const T *X, int ld, int r0, int c0) {
  const int l = lane_id();
  const T *p = X + (r0 + (l & 15)) * ld + c0 + 8 * (l >> 4);
  if constexpr (sizeof(T) == 2) {
    return *(const bf16x8 *)p;
  } else {
    f4 a = *(const f4 *)p, b = *(const f4 *)(p + 4);
    return f8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
}

// Fragment whose reduction index runs down a column (a transposed read):
// lane (g, j) gets X[r0 + 8g + i][c0 + j], i = 0..7.  For bf16 this is two
// gfx950 LDS transpose reads: with lane j of a 16-lane group pointing at
// X[R + j/4][c0 + 4 (j%4)], ds_read_b64_tr_b16 returns X[R + m][c0 + j],
// m = 0..3, to lane j.
template <typename T>
__device__ __forceinline__ frag_t<T> ld_col(const T *X, int ld, int r0, int c0) {
  const int l = lane_id(), g = l >> 4, j = l & 15;
  if constexpr (sizeof(T) == 2) {
    const T *p0 = X + (r0 + 8 * g + (j >> 2)) * ld + c0 + 4 * (j & 3);
    const T *p1 = p0 + 4 * ld;
    s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p0));
    s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(p1));
    s8 r = s8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, r);
  } else {
    const T *p = X + (r0 + 8 * g) * ld + c0 + j;
    f8 r;
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = p[i * ld];
    return r;
  }
}

// B (or A) fragment taken straight from two stacked 16x16 accumulators
// lo = rows [0,16), hi = rows [16,32) of a 32-row slab: lane (g, j) holds
// rows 4g..4g+3 of column j in each, which become slots 0..3 and 4..7.
// The matching operand must list the same 8 indices per lane.
template <typename T> __device__ __forceinline__ frag_t<T> acc_frag(f4 lo, f4 hi) {
  frag_t<T> r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    r[i] = cvt<T>(lo[i]);
    r[4 + i] = cvt<T>(hi[i]);
  }
  return r;
}

// Buffer resource over [base, base + bytes): buffer loads at byte offsets at
// or beyond `bytes` return zeros instead of touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// Clamp a byte count to the 32-bit range of a buffer resource.
__device__ __forceinline__ uint32_t rsrc_bytes(int64_t bytes) {
  return bytes <= 0 ? 0u : (bytes >= 0xFFFFFFF0LL ? 0xFFFFFFF0u : (uint32_t)bytes);
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// Register-staged [ROWS x COLS] tile copy, global -> LDS, for NT threads, with
// compile-time geometry.  init() fixes each thread's byte offsets once (row
// stride gld elements; rows >= rvalid or columns >= cvalid get an offset past
// any buffer, so they read as zero); load() issues the 16-byte buffer loads
// without waiting; store() writes the registers into an LDS tile with leading
// dimension ld.  COLS * sizeof(T) / 16 must be a power of two dividing NT.
template <typename T, int ROWS, int COLS, int NT> struct TileLd {
  static constexpr int EV = 16 / sizeof(T);
  static constexpr int VPR = COLS / EV;
  static constexpr int RSTEP = NT / VPR;
  static constexpr int NV = (ROWS + RSTEP - 1) / RSTEP;
  static_assert(VPR > 0 && (VPR & (VPR - 1)) == 0 && NT % VPR == 0, "tile geometry");
  uint32_t off[NV];
  u32x4 r[NV];
  __device__ __forceinline__ void init(int gld, int rvalid, int cvalid) {
    const int row0 = (int)threadIdx.x / VPR, c = ((int)threadIdx.x % VPR) * EV;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int row = row0 + i * RSTEP;
      const bool ok = row < ROWS && row < rvalid && c < cvalid;
      off[i] = ok ? (uint32_t)(row * gld + c) * (uint32_t)sizeof(T) : 0x80000000u;
    }
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
      r[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off[i], 0, 0));
  }
  // Same, additionally reading columns >= cvalid as zero.
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int cvalid) {
    const bool ok = ((int)threadIdx.x % VPR) * EV < cvalid;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      r[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, ok ? off[i] : 0x80000000u, 0, 0));
  }
  // store() into a tile whose 16-byte chunks are XOR-swizzled per row: chunk
  // c of row r lands at chunk c ^ (((r & 3) << 2) | ((r >> 2) & 3)).
  __device__ __forceinline__ void store_swz(T *dst, int ld) const {
    const int row0 = (int)threadIdx.x / VPR, ch = (int)threadIdx.x % VPR;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int row = row0 + i * RSTEP;
      const int cs = ch ^ (((row & 3) << 2) | ((row >> 2) & 3));
      if (ROWS % RSTEP == 0 || row < ROWS) *(u32x4 *)(dst + row * ld + cs * EV) = r[i];
    }
  }
  // store() into a 2-byte tile whose 8-byte units are XOR-permuted per row:
  // unit u of row r lands at unit u ^ sw(r) (sw(r) below the row's unit count).
  template <typename F> __device__ __forceinline__ void store_xor8(T *dst, int ld, F sw) const {
    static_assert(sizeof(T) == 2, "8-byte units of 2-byte elements");
    const int row0 = (int)threadIdx.x / VPR, ch = (int)threadIdx.x % VPR;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int row = row0 + i * RSTEP;
      const int s = sw(row);
      const u32x4 v = (s & 1) ? u32x4{r[i][2], r[i][3], r[i][0], r[i][1]} : r[i];
      if (ROWS % RSTEP == 0 || row < ROWS) *(u32x4 *)(dst + row * ld + ((ch ^ (s >> 1)) * EV)) = v;
    }
  }
  __device__ __forceinline__ void store(T *dst, int ld) const {
    const int row0 = (int)threadIdx.x / VPR, c = ((int)threadIdx.x % VPR) * EV;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int row = row0 + i * RSTEP;
      if (ROWS % RSTEP == 0 || row < ROWS) *(u32x4 *)(dst + row * ld + c) = r[i];
    }
  }
};

// XCD-aware block mapping: consecutive workgroup ids are dealt round-robin to
// the 8 XCDs, so when the head count is a multiple of 8 the tiles of one head
// are all given ids with the same residue mod 8 (one XCD, one L2), letting
// them share the head's per-chunk operands through that L2.
__device__ __forceinline__ void xcd_map(int nheads, int ntiles, int &head, int &tile) {
  const int id = blockIdx.x;
  if ((nheads & 7) == 0) {
    const int xcd = id & 7, s = id >> 3;
    tile = s % ntiles;
    head = (s / ntiles) * 8 + xcd;
  } else {
    head = id / ntiles;
    tile = id - head * ntiles;
  }
}

}  // namespace gla
