// gla_outgate.hip -- the output side of the GLA layer (Sec. 4.4): each head's
// output row o_t (d_v features) is layer-normalised and gated,
//     y_t = Swish(g_t) (.) (w (.) (o_t - mean) / sqrt(var + eps) + b),
// with g_t the output-gate pre-activation and w, b per-channel affine
// parameters of the concatenated heads ([H][d_v], optional).
//
// Rows are independent and d_v <= 1024, so one wave owns one row at a time:
// lane l holds the EPL consecutive features EPL l .. +EPL-1 in registers (d_v
// is a multiple of 16, so a lane's features are all inside the row or all
// outside it), the row's mean and variance are two-pass wave reductions in
// fp32 (DPP within 16-lane rows, then the four row sums), and every tensor is
// read and written once with one buffer access per lane.  A wave loads a batch
// of consecutive rows of one head before it reduces any of them, so enough
// bytes are in flight to stream at HBM rate; rows and features outside the
// tensors fall outside the buffer ranges (loads give zero, stores drop).
// The backward also forms the per-channel gradients of w and b: each
// workgroup sums its 64 rows' contributions and writes one partial row; a
// second kernel adds the partials of each head in a fixed order.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

constexpr int kOgWaves = 4;        // waves per forward / backward workgroup
constexpr int kOgRowsPerWg = 64;   // rows of one (batch, head) per backward workgroup
constexpr int kOgRedWaves = 16;    // waves per affine-reduction workgroup

// Rows a wave loads per batch: up to 64 bytes of each tensor per lane in the
// forward (two tensors in), half that in the backward (three in, more live).
template <typename T, int EPL>
constexpr int og_rows() {
  return EPL * (int)sizeof(T) >= 64 ? 1 : (EPL * (int)sizeof(T) >= 32 ? 2 : 4);
}
template <typename T, int EPL>
constexpr int og_rows_bwd() {
  return og_rows<T, EPL>() > 1 ? og_rows<T, EPL>() / 2 : 1;
}

struct OgArgs {
  const void *o, *g, *dy;
  const float *w, *b;
  void *y, *d_o, *dg;
  float *stats;        // forward: [rows][2] (mean, rstd), nullable
  float *part;         // backward: [B H tblocks][2][V] partial (dw, db), nullable
  float *dw, *db;      // backward: [H][V], nullable
  int H, T, V, tblocks;
  float eps, inv_v;
};

template <typename T, int EPL>
__device__ __forceinline__ void og_load(__amdgpu_buffer_rsrc_t rs, uint32_t off, float (&x)[EPL]) {
  constexpr int B = EPL * (int)sizeof(T);
  uint32_t r[(B + 3) / 4 < 1 ? 1 : (B + 3) / 4];
  if constexpr (B == 2) {
    r[0] = __builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
  } else if constexpr (B == 4) {
    r[0] = __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
  } else if constexpr (B == 8) {
    const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
    r[0] = v[0];
    r[1] = v[1];
  } else {
#pragma unroll
    for (int c = 0; c < B / 16; ++c) {
      const u32x4 v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * c, 0, 0));
#pragma unroll
      for (int i = 0; i < 4; ++i) r[4 * c + i] = v[i];
    }
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    if constexpr (sizeof(T) == 2) x[i] = __builtin_bit_cast(float, (r[i / 2] >> (16 * (i % 2))) << 16);
    else x[i] = __builtin_bit_cast(float, r[i]);
  }
}

template <typename T, int EPL>
__device__ __forceinline__ void og_store(__amdgpu_buffer_rsrc_t rs, uint32_t off, const float (&x)[EPL]) {
  constexpr int B = EPL * (int)sizeof(T);
  uint32_t r[(B + 3) / 4 < 1 ? 1 : (B + 3) / 4];
#pragma unroll
  for (int i = 0; i < (B + 3) / 4; ++i) r[i] = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    if constexpr (sizeof(T) == 2) {
      const uint32_t h = __builtin_bit_cast(unsigned short, (bf16)x[i]);
      r[i / 2] |= h << (16 * (i % 2));
    } else {
      r[i] = __builtin_bit_cast(uint32_t, x[i]);
    }
  }
  if constexpr (B == 2) {
    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)r[0], rs, off, 0, 0);
  } else if constexpr (B == 4) {
    __builtin_amdgcn_raw_buffer_store_b32(r[0], rs, off, 0, 0);
  } else if constexpr (B == 8) {
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{r[0], r[1]}, rs, off, 0, 0);
  } else {
#pragma unroll
    for (int c = 0; c < B / 16; ++c)
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{r[4 * c], r[4 * c + 1], r[4 * c + 2], r[4 * c + 3]}, rs,
                                             off + 16 * c, 0, 0);
  }
}

// Lane value of the DPP-permuted register (all lanes take part).
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float lane_value(float x, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), lane));
}

// Sum over the wave, the same bits in every lane: a butterfly inside each
// 16-lane row (partners lane^1, lane^2, then the mirrored quad and half row),
// then the four row sums.
__device__ __forceinline__ float wave_sum(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  x += dpp<0x140>(x);  // row_mirror
  return (lane_value(x, 0) + lane_value(x, 16)) + (lane_value(x, 32) + lane_value(x, 48));
}

__device__ __forceinline__ float sigmoid(float x) { return 1.f / (1.f + __expf(-x)); }

// Row statistics of x (lanes past the row hold zeros and are excluded): mean
// and 1 / sqrt(biased variance + eps), the variance taken about the mean.
template <int EPL>
__device__ __forceinline__ void row_stats(const float (&x)[EPL], bool lv, float inv_v, float eps, float &mean,
                                          float &rstd) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i) s += x[i];
  mean = wave_sum(s) * inv_v;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const float d = lv ? x[i] - mean : 0.f;
    q += d * d;
  }
  rstd = rsqrtf(wave_sum(q) * inv_v + eps);
}

// The per-channel affine of head h for this lane's features (1 and 0 when
// absent).
template <int EPL>
__device__ __forceinline__ void load_affine(const OgArgs &a, int h, uint32_t foff, float (&wf)[EPL],
                                            float (&bf)[EPL]) {
  const uint32_t vb = (uint32_t)a.V * 4u;
  if (a.w) {
    og_load<float, EPL>(make_rsrc(a.w + (int64_t)h * a.V, vb), foff, wf);
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) wf[i] = 1.f;
  }
  if (a.b) {
    og_load<float, EPL>(make_rsrc(a.b + (int64_t)h * a.V, vb), foff, bf);
  } else {
#pragma unroll
    for (int i = 0; i < EPL; ++i) bf[i] = 0.f;
  }
}

// Workgroup = (batch-head bh, time block tb) as blockIdx.x = bh tblocks + tb;
// wave w takes the R consecutive rows from (kOgWaves tb + w) R.
template <typename T, int EPL>
__global__ void __launch_bounds__(64 * kOgWaves) outgate_fwd_kernel(OgArgs a) {
  constexpr int R = og_rows<T, EPL>();
  const int w = wave_id(), l = lane_id();
  const int bh = blockIdx.x / a.tblocks, tb = blockIdx.x - bh * a.tblocks;
  const int t0 = (tb * kOgWaves + w) * R;
  if (t0 >= a.T) return;  // whole waves leave together
  const int V = a.V, h = bh % a.H, f0 = EPL * l, nr = min(R, a.T - t0);
  const bool lv = f0 < V;
  constexpr uint32_t esz = sizeof(T);
  const uint32_t rowb = (uint32_t)V * esz, off = lv ? (uint32_t)f0 * esz : 0x80000000u;
  const int64_t base = ((int64_t)bh * a.T + t0) * V;
  const auto ro = make_rsrc((const T *)a.o + base, nr * rowb), rg = make_rsrc((const T *)a.g + base, nr * rowb);
  float x[R][EPL], gg[R][EPL], wf[EPL], bf[EPL];
#pragma unroll
  for (int r = 0; r < R; ++r) og_load<T, EPL>(ro, off + r * rowb, x[r]);
#pragma unroll
  for (int r = 0; r < R; ++r) og_load<T, EPL>(rg, off + r * rowb, gg[r]);
  load_affine<EPL>(a, h, lv ? (uint32_t)f0 * 4u : 0x80000000u, wf, bf);
  const auto ry = make_rsrc((T *)a.y + base, nr * rowb);
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float mean, rstd, y[EPL];
    row_stats<EPL>(x[r], lv, a.inv_v, a.eps, mean, rstd);
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const float ln = (x[r][i] - mean) * rstd * wf[i] + bf[i];
      y[i] = gg[r][i] * sigmoid(gg[r][i]) * ln;
    }
    og_store<T, EPL>(ry, off + r * rowb, y);
    if (a.stats && l == 0 && r < nr) {
      a.stats[2 * ((int64_t)bh * a.T + t0 + r)] = mean;
      a.stats[2 * ((int64_t)bh * a.T + t0 + r) + 1] = rstd;
    }
  }
}

// Workgroup = (batch-head bh, time block tb) as blockIdx.x = bh tblocks + tb:
// rows 64 tb .. +63 of bh, wave w taking 16 consecutive ones in batches of
// R.  Per-lane partial sums of the affine gradients are combined across the
// waves in LDS and written as one partial row.
template <typename T, int EPL>
__global__ void __launch_bounds__(64 * kOgWaves) outgate_bwd_kernel(OgArgs a) {
  constexpr int R = og_rows_bwd<T, EPL>(), RPW = kOgRowsPerWg / kOgWaves;
  __shared__ float sPart[kOgWaves][2][64 * EPL];
  const int w = wave_id(), l = lane_id();
  const int bh = blockIdx.x / a.tblocks, tb = blockIdx.x - bh * a.tblocks;
  const int V = a.V, h = bh % a.H, f0 = EPL * l;
  const bool lv = f0 < V;
  constexpr uint32_t esz = sizeof(T);
  const uint32_t rowb = (uint32_t)V * esz, off = lv ? (uint32_t)f0 * esz : 0x80000000u;
  const int t0 = tb * kOgRowsPerWg + w * RPW, nr = max(0, min(RPW, a.T - t0));
  float wf[EPL], bf[EPL], pw[EPL], pb[EPL];
  load_affine<EPL>(a, h, lv ? (uint32_t)f0 * 4u : 0x80000000u, wf, bf);
#pragma unroll
  for (int i = 0; i < EPL; ++i) pw[i] = pb[i] = 0.f;
  const int64_t base = ((int64_t)bh * a.T + t0) * V;
  // (nr is wave-uniform; readfirstlane keeps the descriptors in SGPRs)
  const uint32_t nb = __builtin_amdgcn_readfirstlane((uint32_t)nr * rowb);
  const auto ro = make_rsrc((const T *)a.o + base, nb), rg = make_rsrc((const T *)a.g + base, nb);
  const auto rdy = make_rsrc((const T *)a.dy + base, nb);
  const auto rdo = make_rsrc((T *)a.d_o + base, nb), rdg = make_rsrc((T *)a.dg + base, nb);
  for (int r0 = 0; r0 < nr; r0 += R) {
    float x[R][EPL], gg[R][EPL], dy[R][EPL];
#pragma unroll
    for (int r = 0; r < R; ++r) og_load<T, EPL>(ro, off + (r0 + r) * rowb, x[r]);
#pragma unroll
    for (int r = 0; r < R; ++r) og_load<T, EPL>(rg, off + (r0 + r) * rowb, gg[r]);
#pragma unroll
    for (int r = 0; r < R; ++r) og_load<T, EPL>(rdy, off + (r0 + r) * rowb, dy[r]);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      // rows past the tensor load as zeros and add nothing to pw, pb
      float mean, rstd;
      row_stats<EPL>(x[r], lv, a.inv_v, a.eps, mean, rstd);
      float xh[EPL], dxh[EPL], dg[EPL], s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        xh[i] = lv ? (x[r][i] - mean) * rstd : 0.f;
        const float sg = sigmoid(gg[r][i]);
        const float ln = xh[i] * wf[i] + bf[i];
        dg[i] = dy[r][i] * ln * (sg * (1.f + gg[r][i] * (1.f - sg)));  // d Swish(g) / dg
        const float dln = dy[r][i] * gg[r][i] * sg;
        pw[i] += dln * xh[i];
        pb[i] += dln;
        dxh[i] = dln * wf[i];
        s1 += dxh[i];
        s2 += dxh[i] * xh[i];
      }
      const float m1 = wave_sum(s1) * a.inv_v, m2 = wave_sum(s2) * a.inv_v;
      float d_o[EPL];
#pragma unroll
      for (int i = 0; i < EPL; ++i) d_o[i] = rstd * (dxh[i] - m1 - xh[i] * m2);
      og_store<T, EPL>(rdo, off + (r0 + r) * rowb, d_o);
      og_store<T, EPL>(rdg, off + (r0 + r) * rowb, dg);
    }
  }
  if (!a.part) return;  // uniform: no affine gradients wanted
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    sPart[w][0][f0 + i] = pw[i];
    sPart[w][1][f0 + i] = pb[i];
  }
  __syncthreads();
  float *dst = a.part + (int64_t)blockIdx.x * 2 * V;
  for (int e = threadIdx.x; e < 2 * V; e += 64 * kOgWaves) {
    const int c = e / V, f = e - c * V;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < kOgWaves; ++q) s += sPart[q][c][f];
    dst[e] = s;
  }
}

// dw[h][f], db[h][f] = sums of the B tblocks partial rows of head h.
// Workgroup = (head h, 64 of the 2V columns) as blockIdx.x = h ncol + col;
// wave w sums partial rows w, w + 16, ... eight loads at a time into four
// accumulators, and the 16 wave sums are added in LDS: a fixed order, so the
// result is reproducible.
__global__ void __launch_bounds__(64 * kOgRedWaves) outgate_affine_kernel(OgArgs a, int B) {
  __shared__ float sRed[kOgRedWaves][64];
  const int ncol = (2 * a.V + 63) / 64;
  const int h = blockIdx.x / ncol, e = (blockIdx.x - h * ncol) * 64 + lane_id(), w = wave_id();
  const int P = B * a.tblocks, V2 = 2 * a.V;
  auto ld = [&](int p) {
    const int b = p / a.tblocks, tb = p - b * a.tblocks;
    return a.part[(((int64_t)b * a.H + h) * a.tblocks + tb) * V2 + e];
  };
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  if (e < V2) {
    int p = w;
    for (; p + 7 * kOgRedWaves < P; p += 8 * kOgRedWaves) {
      float x[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = ld(p + i * kOgRedWaves);
      s0 += x[0] + x[4];
      s1 += x[1] + x[5];
      s2 += x[2] + x[6];
      s3 += x[3] + x[7];
    }
    for (; p < P; p += kOgRedWaves) s0 += ld(p);
  }
  sRed[w][lane_id()] = (s0 + s1) + (s2 + s3);
  __syncthreads();
  if (w != 0 || e >= V2) return;
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < kOgRedWaves; ++q) s += sRed[q][lane_id()];
  const int c = e / a.V, f = e - c * a.V;
  float *dst = c == 0 ? a.dw : a.db;
  if (dst) dst[(int64_t)h * a.V + f] = s;
}

int og_epl(int V) {
  const int e = (V + 63) / 64;
  return e <= 1 ? 1 : (e <= 2 ? 2 : (e <= 4 ? 4 : (e <= 8 ? 8 : 16)));
}

template <typename T, int EPL>
hipError_t og_fwd_t(OgArgs a, int B, hipStream_t st) {
  a.tblocks = (a.T + kOgWaves * og_rows<T, EPL>() - 1) / (kOgWaves * og_rows<T, EPL>());
  hipLaunchKernelGGL((outgate_fwd_kernel<T, EPL>), dim3((unsigned)((int64_t)B * a.H * a.tblocks)),
                     dim3(64 * kOgWaves), 0, st, a);
  return hipGetLastError();
}

hipError_t og_affine(const OgArgs &a, int B, hipStream_t st) {
  const int ncol = (2 * a.V + 63) / 64;
  hipLaunchKernelGGL(outgate_affine_kernel, dim3((unsigned)((int64_t)a.H * ncol)), dim3(64 * kOgRedWaves), 0, st,
                     a, B);
  return hipGetLastError();
}

template <typename T, int EPL>
hipError_t og_bwd_t(const OgArgs &a, int B, hipStream_t st) {
  hipLaunchKernelGGL((outgate_bwd_kernel<T, EPL>), dim3((unsigned)((int64_t)B * a.H * a.tblocks)),
                     dim3(64 * kOgWaves), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !a.part) return e;
  return og_affine(a, B, st);
}

template <typename T>
hipError_t og_dispatch(bool fwd, const OgArgs &a, int B, hipStream_t st) {
  switch (og_epl(a.V)) {
    case 1: return fwd ? og_fwd_t<T, 1>(a, B, st) : og_bwd_t<T, 1>(a, B, st);
    case 2: return fwd ? og_fwd_t<T, 2>(a, B, st) : og_bwd_t<T, 2>(a, B, st);
    case 4: return fwd ? og_fwd_t<T, 4>(a, B, st) : og_bwd_t<T, 4>(a, B, st);
    case 8: return fwd ? og_fwd_t<T, 8>(a, B, st) : og_bwd_t<T, 8>(a, B, st);
    default: return fwd ? og_fwd_t<T, 16>(a, B, st) : og_bwd_t<T, 16>(a, B, st);
  }
}

}  // namespace

size_t outgate_partial_bytes(int B, int H, int T, int V) {
  const int tblocks = (T + kOgRowsPerWg - 1) / kOgRowsPerWg;
  return (size_t)B * H * tblocks * 2 * V * sizeof(float);
}

hipError_t launch_outgate_fwd(int B, int H, int T, int V, int io, const void *o, const void *g, const float *w,
                              const float *b, float eps, void *y, float *stats, hipStream_t st) {
  OgArgs a{};
  a.o = o; a.g = g; a.w = w; a.b = b; a.y = y; a.stats = stats;
  a.H = H; a.T = T; a.V = V; a.eps = eps; a.inv_v = 1.f / (float)V;
  return io == IO_BF16 ? og_dispatch<bf16>(true, a, B, st) : og_dispatch<float>(true, a, B, st);
}

hipError_t launch_outgate_bwd(int B, int H, int T, int V, int io, const void *o, const void *g, const float *w,
                              const float *b, float eps, const void *dy, void *d_o, void *dg, float *dw,
                              float *db, float *part, hipStream_t st) {
  OgArgs a{};
  a.o = o; a.g = g; a.w = w; a.b = b; a.dy = dy; a.d_o = d_o; a.dg = dg; a.dw = dw; a.db = db;
  a.part = (dw || db) ? part : nullptr;
  a.H = H; a.T = T; a.V = V; a.eps = eps; a.inv_v = 1.f / (float)V;
  a.tblocks = (T + kOgRowsPerWg - 1) / kOgRowsPerWg;
  if ((int64_t)B * H * T == 0) {
    // no rows: the affine gradients are sums over nothing
    if (!(dw || db) || H == 0) return hipSuccess;
    return og_affine(a, B, st);  // reads no partials when there are none
  }
  return io == IO_BF16 ? og_dispatch<bf16>(false, a, B, st) : og_dispatch<float>(false, a, B, st);
}

}  // namespace gla
