// gla_launch.hpp -- internal interface between the C-ABI layer and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gla {

enum Io { IO_F32 = 0, IO_BF16 = 1 };

// One validated problem.  N = number of chunks (the last may be shorter).
struct Shape {
  int BH, T, K, V, C, c, N;
  int io;
  float inv_tau;  // 0: the gate argument is log alpha; else 1 / tau of the gate epilogue
  bool sgate;     // scalar gate: one gate value per (head, step), [BH][T]
  int esz() const { return io == IO_BF16 ? 2 : 4; }
  int la_row() const { return sgate ? 1 : K; }  // gate elements per step
};

// Device workspace regions (see gla_api.cpp for the layout).
struct Work {
  void *Qt = nullptr;     // [BH][T][K] io : q (.) Lambda   (Lambda = b_t / b_{chunk start})
  void *Kt = nullptr;     // [BH][T][K] io : k (.) Gamma    (Gamma  = b_{chunk end} / b_t)
  void *P = nullptr;      // [BH][N][C][C] io : intra-chunk matrix, lower triangle
  float *gam = nullptr;   // [BH][N][K] fp32 : chunk decay gamma = b_{chunk end} / b_{chunk start}
  // backward: the dq sweep's hand-offs and the intra-chunk terms (gla_intra.hip)
  float *dP = nullptr;    // [BH][N][C][C] fp32 : (dO V^T) (.) M per chunk, transposed ([s][t])
  void *dki = nullptr;    // [BH][T][K] io : intra-chunk part of dk
  void *dai = nullptr;    // [BH][T][K] io : in-chunk reverse cumsum of q dq_intra - k dk_intra
  float *dat = nullptr;   // [BH][N][K] fp32 : its chunk totals
  float *dqr = nullptr;   // [BH][T][K] fp32 : dq_inter (for dq and the gate gradient in the dk sweep)
  float *cST = nullptr;   // [BH][K] fp32 : rowsum(S_T (.) dS_T) (backward)
  float *dla_part = nullptr;  // [BH][ceil(K/32)][T] fp32 : per key tile sums of the gate
                              //   gradient over its features (scalar gate only)
  // value-side gate of the general form (backward only; E = chunk-local
  // inclusive cumsum of log beta per value column)
  void *Vh = nullptr;         // [BH][T][V] io : V (.) exp(-E)
  void *Oh = nullptr;         // [BH][T][V] io : dO (.) exp(E)
  float *gb = nullptr;        // [BH][N][V] fp32 : chunk decay exp(E_last)
  // sequence segments (few heads, long sequences; the kernels then run on the
  // segmented shape, whose heads are the segments)
  float *Sin = nullptr;       // [BH nseg][K][V] fp32 : each segment's initial state
  float *Sloc = nullptr;      // [BH nseg][K][V] fp32 : local final states; then local dS0
  float *dec = nullptr;       // [BH nseg][K] fp32 : each segment's decay
  float *dSout = nullptr;     // [BH nseg][K][V] fp32 : each segment's final-state gradient
  void *Sb = nullptr;         // chunk-end states S_[n+1] (io), written by the dq sweep (ks_state_bytes)
  float *cpart = nullptr;     // [BH][N][ceil(K/32)][V] fp32 : per key tile colsum(S_[n+1] (.) dS_[n+1])
};

// Returns hipSuccess or the launch error.  Shapes are validated by the caller.
hipError_t launch_prep(const Shape &s, const void *q, const void *k, const void *la,
                       const Work &w, hipStream_t st);
// lb: log beta [BH][T][V] of the value-side gate, nullable (beta = 1)
hipError_t launch_fwd_main(const Shape &s, const void *v, const void *lb, const float *S0, void *o, float *ST,
                           const Work &w, hipStream_t st);
// gb_on: the general form (v, dO are then w.Vh, w.Oh; the states decay by w.gb)
// ng: no gate and no gate gradient wanted (la and the backward's dla NULL)
// The dq sweep: w.dqr (dq_inter), w.dP, w.cST.
hipError_t launch_bwd_dq(const Shape &s, const void *k, const void *la, const void *v,
                         const float *S0, const void *dO, const float *dST,
                         const Work &w, hipStream_t st, bool ng, bool gb_on = false);
// The intra-chunk terms of the backward, after the dq sweep: dq, and w.dki,
// w.dai, w.dat for the dk sweep (w.dki only with ng).
hipError_t launch_bwd_intra(const Shape &s, const void *q, const void *k, const void *la, void *dq, const Work &w,
                            hipStream_t st, bool ng);
hipError_t launch_bwd_dk(const Shape &s, const void *q, const void *k, const void *la,
                         const void *v, const void *dO, const float *dST, const void *dq,
                         void *dk, void *dla, const Work &w, hipStream_t st, bool gb_on = false);
// lb: log beta of the general form (nullable)
hipError_t launch_bwd_dv(const Shape &s, const void *dO, const void *lb, const float *dST, void *dv, float *dS0,
                         const Work &w, hipStream_t st);
// General form, value side: Vh, Oh, gb into w; then (after the sweeps) dlog beta.
hipError_t launch_beta_prep(const Shape &s, const void *v, const void *dO, const void *lb, const Work &w,
                            hipStream_t st);
hipError_t launch_beta_grad(const Shape &s, const void *o, const void *dO, const void *v, const void *dv,
                            void *dlb, const Work &w, hipStream_t st);
size_t ks_state_bytes(const Shape &s);
hipError_t launch_recurrent(const Shape &s, const void *q, const void *k, const void *v,
                            const void *la, const void *lb, const float *S0, void *o, float *ST, hipStream_t st);
// T == 0 edge: S_T = S0 (or 0); dS0 = dS_T (or 0).
hipError_t launch_copy_state(int64_t n, const float *src, float *dst, hipStream_t st);

// Output side (per-head LayerNorm + Swish gate, gla_outgate.hip).
size_t outgate_partial_bytes(int B, int H, int T, int V);
hipError_t launch_outgate_fwd(int B, int H, int T, int V, int io, const void *o, const void *g, const float *w,
                              const float *b, float eps, void *y, float *stats, hipStream_t st);
hipError_t launch_outgate_bwd(int B, int H, int T, int V, int io, const void *o, const void *g, const float *w,
                              const float *b, float eps, const void *dy, void *d_o, void *dg, float *dw,
                              float *db, float *part, hipStream_t st);

// Sequence segments (gla_segment.hip); s2 is the segmented shape.
hipError_t launch_seg_decay(const Shape &s2, const float *gam, float *dec, hipStream_t st);
hipError_t launch_seg_fwd_scan(int BH, int nseg, int K, int V, const float *dec, const float *S0, const float *Sloc,
                               float *Sin, float *ST, hipStream_t st);
hipError_t launch_seg_bwd_scan(int BH, int nseg, int K, int V, const float *dec, const float *dST,
                               const float *dS0loc, float *dSout, float *dS0, hipStream_t st);
// LDS bytes each kernel needs (0 means the shape is not supported).
size_t lds_prep(const Shape &s);
size_t lds_fwd_main(const Shape &s);
size_t lds_bwd_intra(const Shape &s);
size_t lds_bwd_dq(const Shape &s);
size_t lds_bwd_dk(const Shape &s);
size_t lds_bwd_dv(const Shape &s);

constexpr size_t kMaxLds = 160 * 1024;

}  // namespace gla
