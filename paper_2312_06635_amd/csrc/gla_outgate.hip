// gla_outgate.hip -- the output side of the GLA layer (Sec. 4.4): each head's
// output row o_t (d_v features) is layer-normalised and gated,
//     y_t = Swish(g_t) (.) (w (.) (o_t - mean) / sqrt(var + eps) + b),
// with g_t the output-gate pre-activation and w, b per-channel affine
// parameters of the concatenated heads ([H][d_v], optional).
//
// Rows are independent and d_v <= 1024, so one wave owns one row: lane l
// holds the EPL consecutive features EPL l .. +EPL-1 in registers, the row's
// mean and variance are two-pass wave reductions in fp32, and every tensor is
// read and written once with one buffer access per lane (rows and features
// outside the tensors fall outside the buffer ranges).  The backward also
// forms the per-channel gradients of w and b: each workgroup sums its rows'
// contributions (one head, 64 consecutive time steps) and writes one partial
// row; a second kernel adds the partials of each head in a fixed order.
#include "gla_common.hpp"
#include "gla_launch.hpp"

namespace gla {

namespace {

constexpr int kOgWaves = 4;      // rows in flight per workgroup
constexpr int kOgRowsPerWg = 64; // rows of one (batch, head) per backward workgroup

struct OgArgs {
  const void *o, *g, *dy;
  const float *w, *b;
  void *y, *d_o, *dg;
  float *stats;        // forward: [rows][2] (mean, rstd), nullable
  float *part;         // backward: [nwg][2][V] partial (dw, db), nullable
  float *dw, *db;      // backward: [H][V], nullable
  int H, T, V, rows, tblocks;
  float eps;
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

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

__device__ __forceinline__ float sigmoid(float x) { return 1.f / (1.f + __expf(-x)); }

// Row statistics of x (features beyond V are zero and excluded): mean and
// 1 / sqrt(biased variance + eps), the variance taken about the mean.
template <int EPL>
__device__ __forceinline__ void row_stats(const float (&x)[EPL], bool (&in)[EPL], int V, float eps, float &mean,
                                          float &rstd) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i) s += x[i];
  mean = wave_sum(s) / (float)V;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const float d = in[i] ? x[i] - mean : 0.f;
    q += d * d;
  }
  rstd = rsqrtf(wave_sum(q) / (float)V + eps);
}

template <typename T, int EPL>
__global__ void __launch_bounds__(64 * kOgWaves) outgate_fwd_kernel(OgArgs a) {
  const int w = wave_id(), l = lane_id();
  const int row = blockIdx.x * kOgWaves + w;
  if (row >= a.rows) return;  // whole waves leave together
  const int V = a.V, h = (row / a.T) % a.H, f0 = EPL * l;
  const int esz = sizeof(T);
  const uint32_t rb = (uint32_t)(V * esz);
  const uint32_t off = f0 < V ? (uint32_t)(f0 * esz) : 0x80000000u;
  const int64_t base = (int64_t)row * V;
  float x[EPL], gg[EPL];
  bool in[EPL];
  og_load<T, EPL>(make_rsrc((const T *)a.o + base, rb), off, x);
  og_load<T, EPL>(make_rsrc((const T *)a.g + base, rb), off, gg);
#pragma unroll
  for (int i = 0; i < EPL; ++i) in[i] = f0 + i < V;
  float mean, rstd;
  row_stats<EPL>(x, in, V, a.eps, mean, rstd);
  float y[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int f = f0 + i;
    const float wf = (a.w && in[i]) ? a.w[h * V + f] : 1.f;
    const float bf = (a.b && in[i]) ? a.b[h * V + f] : 0.f;
    const float ln = (x[i] - mean) * rstd * wf + bf;
    y[i] = gg[i] * sigmoid(gg[i]) * ln;
  }
  og_store<T, EPL>(make_rsrc((T *)a.y + base, rb), off, y);
  if (a.stats && l == 0) {
    a.stats[2 * (int64_t)row] = mean;
    a.stats[2 * (int64_t)row + 1] = rstd;
  }
}

// Workgroup (time block tb, batch-head bh): rows bh T + 64 tb .. +63, wave w
// taking every fourth.  Per-lane partial sums of the affine gradients are
// combined across the waves in LDS and written as one partial row.
template <typename T, int EPL>
__global__ void __launch_bounds__(64 * kOgWaves) outgate_bwd_kernel(OgArgs a) {
  __shared__ float sPart[kOgWaves][2][64 * EPL];
  const int w = wave_id(), l = lane_id();
  const int tb = blockIdx.x, bh = blockIdx.y;
  const int V = a.V, h = bh % a.H, f0 = EPL * l;
  const int esz = sizeof(T);
  const uint32_t rb = (uint32_t)(V * esz);
  const uint32_t off = f0 < V ? (uint32_t)(f0 * esz) : 0x80000000u;
  bool in[EPL];
  float wf[EPL], bf[EPL], pw[EPL], pb[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    in[i] = f0 + i < V;
    wf[i] = (a.w && in[i]) ? a.w[h * V + f0 + i] : 1.f;
    bf[i] = (a.b && in[i]) ? a.b[h * V + f0 + i] : 0.f;
    pw[i] = pb[i] = 0.f;
  }
  const int t_end = min(a.T, kOgRowsPerWg * (tb + 1));
  for (int t = kOgRowsPerWg * tb + w; t < t_end; t += kOgWaves) {
    const int64_t base = ((int64_t)bh * a.T + t) * V;
    float x[EPL], gg[EPL], dy[EPL];
    og_load<T, EPL>(make_rsrc((const T *)a.o + base, rb), off, x);
    og_load<T, EPL>(make_rsrc((const T *)a.g + base, rb), off, gg);
    og_load<T, EPL>(make_rsrc((const T *)a.dy + base, rb), off, dy);
    float mean, rstd;
    row_stats<EPL>(x, in, V, a.eps, mean, rstd);
    float xh[EPL], dxh[EPL], dg[EPL], s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      xh[i] = in[i] ? (x[i] - mean) * rstd : 0.f;
      const float sg = sigmoid(gg[i]);
      const float r = gg[i] * sg;
      const float ln = xh[i] * wf[i] + bf[i];
      dg[i] = dy[i] * ln * (sg * (1.f + gg[i] * (1.f - sg)));  // d Swish(g) / dg
      const float dln = dy[i] * r;
      pw[i] += dln * xh[i];
      pb[i] += dln;
      dxh[i] = dln * wf[i];
      s1 += dxh[i];
      s2 += dxh[i] * xh[i];
    }
    const float m1 = wave_sum(s1) / (float)V, m2 = wave_sum(s2) / (float)V;
    float d_o[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) d_o[i] = rstd * (dxh[i] - m1 - xh[i] * m2);
    og_store<T, EPL>(make_rsrc((T *)a.d_o + base, rb), off, d_o);
    og_store<T, EPL>(make_rsrc((T *)a.dg + base, rb), off, dg);
  }
  if (!a.part) return;  // uniform: no affine gradients wanted
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    sPart[w][0][f0 + i] = pw[i];
    sPart[w][1][f0 + i] = pb[i];
  }
  __syncthreads();
  float *dst = a.part + ((int64_t)bh * a.tblocks + tb) * 2 * V;
  for (int e = threadIdx.x; e < 2 * V; e += 64 * kOgWaves) {
    const int c = e / V, f = e - c * V;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < kOgWaves; ++q) s += sPart[q][c][f];
    dst[e] = s;
  }
}

// dw[h][f], db[h][f] = sums of the partial rows of head h over batch rows and
// time blocks, in a fixed order.
__global__ void __launch_bounds__(256) outgate_affine_kernel(OgArgs a, int B) {
  const int h = blockIdx.y, e = blockIdx.x * 256 + threadIdx.x;
  if (e >= 2 * a.V) return;
  float s = 0.f;
  for (int b = 0; b < B; ++b) {
    const float *p = a.part + ((int64_t)(b * a.H + h) * a.tblocks) * 2 * a.V + e;
    for (int tb = 0; tb < a.tblocks; ++tb) s += p[(int64_t)tb * 2 * a.V];
  }
  const int c = e / a.V, f = e - c * a.V;
  float *dst = c == 0 ? a.dw : a.db;
  if (dst) dst[h * a.V + f] = s;
}

int og_epl(int V) {
  const int e = (V + 63) / 64;
  return e <= 1 ? 1 : (e <= 2 ? 2 : (e <= 4 ? 4 : (e <= 8 ? 8 : 16)));
}

template <typename T, int EPL>
hipError_t og_fwd_t(const OgArgs &a, hipStream_t st) {
  hipLaunchKernelGGL((outgate_fwd_kernel<T, EPL>), dim3((a.rows + kOgWaves - 1) / kOgWaves), dim3(64 * kOgWaves),
                     0, st, a);
  return hipGetLastError();
}

template <typename T, int EPL>
hipError_t og_bwd_t(const OgArgs &a, int B, hipStream_t st) {
  hipLaunchKernelGGL((outgate_bwd_kernel<T, EPL>), dim3(a.tblocks, B * a.H), dim3(64 * kOgWaves), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !a.part) return e;
  hipLaunchKernelGGL(outgate_affine_kernel, dim3((2 * a.V + 255) / 256, a.H), dim3(256), 0, st, a, B);
  return hipGetLastError();
}

template <typename T>
hipError_t og_dispatch(bool fwd, const OgArgs &a, int B, hipStream_t st) {
  switch (og_epl(a.V)) {
    case 1: return fwd ? og_fwd_t<T, 1>(a, st) : og_bwd_t<T, 1>(a, B, st);
    case 2: return fwd ? og_fwd_t<T, 2>(a, st) : og_bwd_t<T, 2>(a, B, st);
    case 4: return fwd ? og_fwd_t<T, 4>(a, st) : og_bwd_t<T, 4>(a, B, st);
    case 8: return fwd ? og_fwd_t<T, 8>(a, st) : og_bwd_t<T, 8>(a, B, st);
    default: return fwd ? og_fwd_t<T, 16>(a, st) : og_bwd_t<T, 16>(a, B, st);
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
  a.H = H; a.T = T; a.V = V; a.rows = B * H * T; a.eps = eps;
  return io == IO_BF16 ? og_dispatch<bf16>(true, a, B, st) : og_dispatch<float>(true, a, B, st);
}

hipError_t launch_outgate_bwd(int B, int H, int T, int V, int io, const void *o, const void *g, const float *w,
                              const float *b, float eps, const void *dy, void *d_o, void *dg, float *dw,
                              float *db, float *part, hipStream_t st) {
  OgArgs a{};
  a.o = o; a.g = g; a.w = w; a.b = b; a.dy = dy; a.d_o = d_o; a.dg = dg; a.dw = dw; a.db = db;
  a.part = (dw || db) ? part : nullptr;
  a.H = H; a.T = T; a.V = V; a.rows = B * H * T; a.eps = eps;
  a.tblocks = (T + kOgRowsPerWg - 1) / kOgRowsPerWg;
  if (a.rows == 0) {
    // no rows: the affine gradients are sums over nothing
    if (!a.part || H == 0) return hipSuccess;
    hipLaunchKernelGGL(outgate_affine_kernel, dim3((2 * V + 255) / 256, H), dim3(256), 0, st, a, B);
    return hipGetLastError();
  }
  return io == IO_BF16 ? og_dispatch<bf16>(false, a, B, st) : og_dispatch<float>(false, a, B, st);
}

}  // namespace gla
