// gla_api.cpp -- the C ABI declared in include/gla.h: argument validation,
// workspace layout and kernel sequencing.  No device memory is allocated here.
#include "gla.h"

#include <hip/hip_runtime.h>

#include "gla_launch.hpp"

#define GLA_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

using gla::Shape;
using gla::Work;

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Validates the problem and fills the internal shape.  The rules are the
// supported-shape list of include/gla.h.  chunked: a chunkwise call (the
// recurrent calls have no chunk grid, so no limit on the chunk count).
gla_status make_shape(const gla_problem *p, Shape &s, bool chunked = true) {
  if (!p) return GLA_ERR_NULL;
  if (p->io != GLA_F32 && p->io != GLA_BF16) return GLA_ERR_DTYPE;
  if (p->B < 0 || p->H < 0 || p->T < 0 || p->dk <= 0 || p->dv <= 0 || p->chunk <= 0 ||
      p->subchunk <= 0)
    return GLA_ERR_SHAPE;
  if (p->chunk % p->subchunk != 0) return GLA_ERR_SHAPE;
  if (p->dk % 16 != 0 || p->dv % 16 != 0 || p->dk > 256 || p->dv > 1024) return GLA_ERR_UNSUPPORTED;
  if (p->chunk != 16 && p->chunk != 32 && p->chunk != 64) return GLA_ERR_UNSUPPORTED;
  if (16 % p->subchunk != 0) return GLA_ERR_UNSUPPORTED;
  const int64_t BH = (int64_t)p->B * p->H;
  if (BH > 65535) return GLA_ERR_UNSUPPORTED;  // heads are a grid dimension of the prep and recurrent kernels
  s.BH = (int)BH;
  s.T = p->T;
  s.K = p->dk;
  s.V = p->dv;
  s.C = p->chunk;
  s.c = p->subchunk;
  s.N = (p->T + p->chunk - 1) / p->chunk;
  s.io = p->io == GLA_BF16 ? gla::IO_BF16 : gla::IO_F32;
  // gate_tau: 0 (the gate argument is log alpha) or a finite tau > 0
  if (!(p->gate_tau == 0.f || (p->gate_tau > 0.f && p->gate_tau < 3.0e38f))) return GLA_ERR_SHAPE;
  s.inv_tau = p->gate_tau == 0.f ? 0.f : 1.f / p->gate_tau;
  s.sgate = (p->flags & GLA_FLAG_SCALAR_GATE) != 0;
  if (chunked && s.N > 65535) return GLA_ERR_UNSUPPORTED;  // chunks are a grid dimension
  // one head's rows of any tensor must span less than 2 GiB (32-bit buffer offsets)
  const int64_t wmax = p->dk > p->dv ? p->dk : p->dv;
  // (fp32 workspace rows included: 4 bytes per element)
  if ((int64_t)p->T * wmax * 4 >= (int64_t)1 << 31) return GLA_ERR_UNSUPPORTED;
  return GLA_OK;
}

// A kernel's LDS need of 0 means it has no variant for the shape.
bool lds_bad(size_t bytes) { return bytes == 0 || bytes > gla::kMaxLds; }

gla_status check_lds(const Shape &s, bool bwd) {
  if (lds_bad(gla::lds_prep(s)) || lds_bad(gla::lds_fwd_main(s))) return GLA_ERR_UNSUPPORTED;
  if (bwd && (lds_bad(gla::lds_bwd_intra(s)) || lds_bad(gla::lds_bwd_dq(s)) || lds_bad(gla::lds_bwd_dk(s)) ||
              lds_bad(gla::lds_bwd_dv(s))))
    return GLA_ERR_UNSUPPORTED;
  return GLA_OK;
}

// Sequence segments: with few heads and long sequences, each head's
// sequence is split into nseg segments of whole chunks (at least four each),
// processed as separate heads and joined by the segment scans of
// gla_segment.hip (App. A.2's two-stage form).  nseg minimises a simple cost:
// the chunks each sweep walks in sequence times the rounds of 256 workgroups
// it needs (key sweeps weighted 2 against 1 for the value sweeps, which run
// twice when segmented); ties keep fewer segments.  Decided from the shape
// alone, so forward and backward agree.  The general form (value-side gate)
// is not segmented.
int choose_nseg(const Shape &s) {
  if (s.T <= 0 || s.T % s.C != 0) return 1;
  const int64_t KT = (s.K + 31) / 32, VT = (s.V + 63) / 64;
  auto rounds = [](int64_t wgs) { return (wgs + 255) / 256; };
  auto cost = [&](int n) {
    const int64_t steps = s.N / n;
    return 4 * rounds((int64_t)s.BH * n * KT) * steps + (n > 1 ? 4 : 2) * rounds((int64_t)s.BH * n * VT) * steps;
  };
  int best = 1;
  int64_t best_cost = cost(1);
  for (int n = 2; s.N % n == 0 && s.N / n >= 4 && (int64_t)s.BH * n <= 65535; n *= 2) {
    const int64_t c = cost(n);
    if (c < best_cost) {
      best = n;
      best_cost = c;
    }
  }
  return best;
}

// The segment count a call runs with: the caller's (GLA_SEGMENTS), else the
// cost model's; 0 when the caller's does not fit the shape.  general: the
// value-gate calls, which run unsegmented.
int resolve_nseg(const Shape &s, uint32_t flags, bool general) {
  const int want = (int)((flags & GLA_SEGMENTS_MASK) >> GLA_SEGMENTS_SHIFT);
  if (want == 0) return general ? 1 : choose_nseg(s);
  if (want == 1 || (s.T == 0 && !general)) return 1;
  if (general || s.T % s.C != 0 || s.N % want != 0 || (int64_t)s.BH * want > 65535) return 0;
  return want;
}

Shape seg_shape(const Shape &s, int nseg) {
  Shape t = s;
  t.BH = s.BH * nseg;
  t.T = s.T / nseg;
  t.N = s.N / nseg;
  return t;
}

// Workspace layout of the (segmented) shape s; op 1 extends op 0, op 2 (the
// general form's backward) extends op 1.  Returns the total byte count and, if
// base is non-null, the region pointers.
size_t layout(const Shape &s, int op, char *base, Work *w, int nseg) {
  const size_t es = s.esz();
  const size_t rows = (size_t)s.BH * s.T, chunks = (size_t)s.BH * s.N;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return base ? (void *)(base + at) : nullptr;
  };
  void *Qt = take(rows * s.K * es);
  void *Kt = take(rows * s.K * es);
  void *P = take(chunks * s.C * s.C * es);
  void *gam = take(chunks * s.K * sizeof(float));
  const size_t states = (size_t)s.BH * s.K * s.V * sizeof(float);  // s.BH counts the segments
  void *Sin = nullptr, *Sloc = nullptr, *dec = nullptr, *dSout = nullptr;
  if (nseg > 1) {
    Sin = take(states);
    Sloc = take(states);
    dec = take((size_t)s.BH * s.K * sizeof(float));
  }
  void *dP = nullptr, *dki = nullptr, *dai = nullptr, *dat = nullptr, *dqr = nullptr;
  void *cST = nullptr, *dla_part = nullptr;
  void *Vh = nullptr, *Oh = nullptr, *gb = nullptr, *Sb = nullptr, *cpart = nullptr;
  if (op >= 1) {
    dP = take(chunks * s.C * s.C * sizeof(float));
    dki = take(rows * s.K * es);
    dai = take(rows * s.K * es);
    dat = take(chunks * s.K * sizeof(float));
    dqr = take(rows * s.K * sizeof(float));
    cST = take((size_t)s.BH * s.K * sizeof(float));
    if (s.sgate) dla_part = take(rows * ((s.K + 31) / 32) * sizeof(float));
    if (nseg > 1) dSout = take(states);
  }
  if (op == 2) {
    Vh = take(rows * s.V * es);
    Oh = take(rows * s.V * es);
    gb = take(chunks * s.V * sizeof(float));
    Sb = take(gla::ks_state_bytes(s));
    cpart = take(chunks * ((s.K + 31) / 32) * s.V * sizeof(float));
  }
  if (w) {
    w->Qt = Qt; w->Kt = Kt; w->P = P; w->gam = (float *)gam;
    w->dP = (float *)dP; w->dki = dki; w->dai = dai; w->dat = (float *)dat; w->dqr = (float *)dqr;
    w->cST = (float *)cST; w->dla_part = (float *)dla_part;
    w->Vh = Vh; w->Oh = Oh; w->gb = (float *)gb; w->Sb = Sb; w->cpart = (float *)cpart;
    w->Sin = (float *)Sin; w->Sloc = (float *)Sloc; w->dec = (float *)dec; w->dSout = (float *)dSout;
  }
  return off;
}

gla_status hip_status(hipError_t e) { return e == hipSuccess ? GLA_OK : GLA_ERR_HIP; }

// Without a gate the gated operands Q (.) Lambda, K (.) Gamma are q and k
// themselves: the kernels read the inputs in their place (the prep kernel
// then does not write them).
void alias_ungated(Work &w, const void *log_alpha, const void *q, const void *k) {
  if (log_alpha) return;
  w.Qt = const_cast<void *>(q);
  w.Kt = const_cast<void *>(k);
}

}  // namespace

GLA_EXPORT const char *gla_status_string(gla_status st) {
  switch (st) {
    case GLA_OK: return "GLA_OK";
    case GLA_ERR_NULL: return "GLA_ERR_NULL: a required pointer is NULL";
    case GLA_ERR_SHAPE: return "GLA_ERR_SHAPE: a dimension is negative or inconsistent";
    case GLA_ERR_DTYPE: return "GLA_ERR_DTYPE: unknown io dtype";
    case GLA_ERR_UNSUPPORTED: return "GLA_ERR_UNSUPPORTED: shape outside what the kernels implement";
    case GLA_ERR_WORKSPACE: return "GLA_ERR_WORKSPACE: workspace NULL or too small";
    case GLA_ERR_HIP: return "GLA_ERR_HIP: a HIP call or kernel launch failed";
    case GLA_ERR_SCRATCH: return "GLA_ERR_SCRATCH: the problem's workspace exceeds the fixed scratch array";
  }
  return "GLA_ERR_UNKNOWN";
}

GLA_EXPORT size_t gla_workspace_bytes(const gla_problem *prob, int op) {
  Shape s;
  if (make_shape(prob, s) != GLA_OK || op < 0 || op > 2) return 0;
  const int nseg = resolve_nseg(s, prob->flags, op == 2);
  if (nseg == 0) return 0;
  return layout(seg_shape(s, nseg), op, nullptr, nullptr, nseg);
}

namespace {

gla_status chunk_fwd(const gla_problem *prob, const void *q, const void *k, const void *v,
                     const void *log_alpha, const void *log_beta, const float *S0, void *o, float *S_T,
                     void *workspace, size_t workspace_bytes, void *stream) {
  Shape s;
  gla_status st = make_shape(prob, s);
  if (st != GLA_OK) return st;
  if (!log_alpha) s.inv_tau = 0.f;  // no gate: alpha = 1 whatever gate_tau says
  if ((st = check_lds(s, false)) != GLA_OK) return st;
  const unsigned stage = (prob->flags & GLA_STAGE_MASK) >> GLA_STAGE_SHIFT;
  if (stage > 2) return GLA_ERR_SHAPE;
  const bool any = (int64_t)s.BH * s.T > 0;
  if (any && (!q || !k || !v || !o)) return GLA_ERR_NULL;
  const int nseg = resolve_nseg(s, prob->flags, log_beta != nullptr);
  if (nseg == 0) return GLA_ERR_UNSUPPORTED;
  const Shape s2 = seg_shape(s, nseg);
  const size_t need = layout(s2, 0, nullptr, nullptr, nseg);
  if (any && (!workspace || workspace_bytes < need)) return GLA_ERR_WORKSPACE;
  hipStream_t hs = (hipStream_t)stream;
  if (s.BH == 0) return GLA_OK;
  if (s.T == 0)
    return hip_status(gla::launch_copy_state((int64_t)s.BH * s.K * s.V, S0, S_T, hs));
  Work w;
  layout(s2, 0, (char *)workspace, &w, nseg);
  alias_ungated(w, log_alpha, q, k);
  hipError_t e = hipSuccess;
  if (stage == 0 || stage == 1) e = gla::launch_prep(s2, q, k, log_alpha, w, hs);
  if (e == hipSuccess && (stage == 0 || stage == 2)) {
    if (nseg == 1) {
      e = gla::launch_fwd_main(s, v, log_beta, S0, o, S_T, w, hs);
    } else {
      // local final states, the segment scan, then the outputs from each
      // segment's true initial state
      e = gla::launch_fwd_main(s2, v, nullptr, nullptr, o, w.Sloc, w, hs);
      if (e == hipSuccess) e = gla::launch_seg_decay(s2, w.gam, w.dec, hs);
      if (e == hipSuccess) e = gla::launch_seg_fwd_scan(s.BH, nseg, s.K, s.V, w.dec, S0, w.Sloc, w.Sin, S_T, hs);
      if (e == hipSuccess) e = gla::launch_fwd_main(s2, v, nullptr, w.Sin, o, nullptr, w, hs);
    }
  }
  return hip_status(e);
}

gla_status recurrent_fwd(const gla_problem *prob, const void *q, const void *k, const void *v,
                         const void *log_alpha, const void *log_beta, const float *S0, void *o, float *S_T,
                         void *stream) {
  if (!prob) return GLA_ERR_NULL;
  gla_problem p = *prob;
  p.chunk = 16;  // the recurrent form ignores the chunk fields
  p.subchunk = 16;
  Shape s;
  gla_status st = make_shape(&p, s, false);
  if (st != GLA_OK) return st;
  if (!log_alpha) s.inv_tau = 0.f;  // no gate: alpha = 1 whatever gate_tau says
  const bool any = (int64_t)s.BH * s.T > 0;
  if (any && (!q || !k || !v || !o)) return GLA_ERR_NULL;
  hipStream_t hs = (hipStream_t)stream;
  if (s.BH == 0) return GLA_OK;
  if (s.T == 0)
    return hip_status(gla::launch_copy_state((int64_t)s.BH * s.K * s.V, S0, S_T, hs));
  return hip_status(gla::launch_recurrent(s, q, k, v, log_alpha, log_beta, S0, o, S_T, hs));
}

}  // namespace

GLA_EXPORT gla_status gla_chunk_fwd(const gla_problem *prob, const void *q, const void *k,
                                    const void *v, const void *log_alpha, const float *S0,
                                    void *o, float *S_T, void *workspace, size_t workspace_bytes,
                                    void *stream) {
  return chunk_fwd(prob, q, k, v, log_alpha, nullptr, S0, o, S_T, workspace, workspace_bytes, stream);
}

GLA_EXPORT gla_status gla_chunk_fwd_general(const gla_problem *prob, const void *q, const void *k,
                                            const void *v, const void *log_alpha, const void *log_beta,
                                            const float *S0, void *o, float *S_T, void *workspace,
                                            size_t workspace_bytes, void *stream) {
  return chunk_fwd(prob, q, k, v, log_alpha, log_beta, S0, o, S_T, workspace, workspace_bytes, stream);
}

GLA_EXPORT gla_status gla_chunk_bwd(const gla_problem *prob, const void *q, const void *k,
                                    const void *v, const void *log_alpha, const float *S0,
                                    const void *dO, const float *dS_T, void *dq, void *dk,
                                    void *dv, void *dlog_alpha, float *dS0, void *workspace,
                                    size_t workspace_bytes, void *stream) {
  Shape s;
  gla_status st = make_shape(prob, s);
  if (st != GLA_OK) return st;
  if (!log_alpha) s.inv_tau = 0.f;  // no gate: alpha = 1 whatever gate_tau says
  if ((st = check_lds(s, true)) != GLA_OK) return st;
  const unsigned stage = (prob->flags & GLA_STAGE_MASK) >> GLA_STAGE_SHIFT;
  if (stage > 5) return GLA_ERR_SHAPE;
  const bool any = (int64_t)s.BH * s.T > 0;
  if (any && (!q || !k || !v || !dO || !dq || !dk || !dv)) return GLA_ERR_NULL;
  const int nseg = resolve_nseg(s, prob->flags, false);
  if (nseg == 0) return GLA_ERR_UNSUPPORTED;
  const Shape s2 = seg_shape(s, nseg);
  const size_t need = layout(s2, 1, nullptr, nullptr, nseg);
  if (any && (!workspace || workspace_bytes < need)) return GLA_ERR_WORKSPACE;
  hipStream_t hs = (hipStream_t)stream;
  if (s.BH == 0) return GLA_OK;
  if (s.T == 0)
    return hip_status(gla::launch_copy_state((int64_t)s.BH * s.K * s.V, dS_T, dS0, hs));
  auto run = [stage](unsigned k) { return stage == 0 || stage == k; };
  // no gate and no gate gradient: the kernels' alpha = 1 variants
  const bool ng = !log_alpha && !dlog_alpha;
  Work w;
  layout(s2, 1, (char *)workspace, &w, nseg);
  alias_ungated(w, log_alpha, q, k);
  hipError_t e = hipSuccess;
  if (run(1) && !(prob->flags & GLA_FLAG_REUSE_FWD_WORKSPACE)) {
    e = gla::launch_prep(s2, q, k, log_alpha, w, hs);
    if (nseg > 1) {
      // each segment's initial state, as in the forward (dv serves as scratch
      // for the outputs, which are not needed here)
      if (e == hipSuccess) e = gla::launch_fwd_main(s2, v, nullptr, nullptr, dv, w.Sloc, w, hs);
      if (e == hipSuccess) e = gla::launch_seg_decay(s2, w.gam, w.dec, hs);
      if (e == hipSuccess) e = gla::launch_seg_fwd_scan(s.BH, nseg, s.K, s.V, w.dec, S0, w.Sloc, w.Sin, nullptr, hs);
    }
  }
  // per segment: initial state and final-state gradient (the head's own S0
  // and dS_T when unsegmented)
  const float *S0s = nseg > 1 ? w.Sin : S0, *dSTs = nseg > 1 ? w.dSout : dS_T;
  if (e == hipSuccess && run(2)) {
    if (nseg > 1) {
      // local initial-state gradients from a zero final-state gradient, then
      // the reverse segment scan (which also gives the head's dS0)
      e = gla::launch_bwd_dv(s2, dO, nullptr, nullptr, dv, w.Sloc, w, hs);
      if (e == hipSuccess)
        e = gla::launch_seg_bwd_scan(s.BH, nseg, s.K, s.V, w.dec, dS_T, w.Sloc, w.dSout, dS0, hs);
    }
    if (e == hipSuccess) e = gla::launch_bwd_dq(s2, k, log_alpha, v, S0s, dO, dSTs, w, hs, ng);
  }
  if (e == hipSuccess && run(3)) e = gla::launch_bwd_intra(s2, q, k, log_alpha, dq, w, hs, ng);
  if (e == hipSuccess && run(4))
    e = gla::launch_bwd_dk(s2, q, k, log_alpha, v, dO, dSTs, dq, dk, dlog_alpha, w, hs);
  if (e == hipSuccess && run(5)) e = gla::launch_bwd_dv(s2, dO, nullptr, dSTs, dv, nseg > 1 ? nullptr : dS0, w, hs);
  return hip_status(e);
}

GLA_EXPORT gla_status gla_chunk_bwd_general(const gla_problem *prob, const void *q, const void *k,
                                            const void *v, const void *log_alpha, const void *log_beta,
                                            const float *S0, const void *o, const void *dO, const float *dS_T,
                                            void *dq, void *dk, void *dv, void *dlog_alpha, void *dlog_beta,
                                            float *dS0, void *workspace, size_t workspace_bytes, void *stream) {
  Shape s;
  gla_status st = make_shape(prob, s);
  if (st != GLA_OK) return st;
  if (!log_alpha) s.inv_tau = 0.f;
  if (s.inv_tau != 0.f) return GLA_ERR_UNSUPPORTED;  // no key-gate epilogue with the value-side gate
  if ((st = check_lds(s, true)) != GLA_OK) return st;
  const unsigned stage = (prob->flags & GLA_STAGE_MASK) >> GLA_STAGE_SHIFT;
  if (stage > 7) return GLA_ERR_SHAPE;
  const bool any = (int64_t)s.BH * s.T > 0;
  if (any && (!q || !k || !v || !log_beta || !dO || !dq || !dk || !dv)) return GLA_ERR_NULL;
  if (any && dlog_beta && !o) return GLA_ERR_NULL;
  if (resolve_nseg(s, prob->flags, true) != 1) return GLA_ERR_UNSUPPORTED;
  const size_t need = layout(s, 2, nullptr, nullptr, 1);
  if (any && (!workspace || workspace_bytes < need)) return GLA_ERR_WORKSPACE;
  hipStream_t hs = (hipStream_t)stream;
  if (s.BH == 0) return GLA_OK;
  if (s.T == 0)
    return hip_status(gla::launch_copy_state((int64_t)s.BH * s.K * s.V, dS_T, dS0, hs));
  auto run = [stage](unsigned k) { return stage == 0 || stage == k; };
  Work w;
  layout(s, 2, (char *)workspace, &w, 1);
  alias_ungated(w, log_alpha, q, k);
  hipError_t e = hipSuccess;
  if (run(1) && !(prob->flags & GLA_FLAG_REUSE_FWD_WORKSPACE))
    e = gla::launch_prep(s, q, k, log_alpha, w, hs);
  if (e == hipSuccess && run(2)) e = gla::launch_beta_prep(s, v, dO, log_beta, w, hs);
  if (e == hipSuccess && run(3)) e = gla::launch_bwd_dq(s, k, log_alpha, w.Vh, S0, w.Oh, dS_T, w, hs, false, true);
  if (e == hipSuccess && run(4)) e = gla::launch_bwd_intra(s, q, k, log_alpha, dq, w, hs, false);
  if (e == hipSuccess && run(5))
    e = gla::launch_bwd_dk(s, q, k, log_alpha, w.Vh, w.Oh, dS_T, dq, dk, dlog_alpha, w, hs, true);
  if (e == hipSuccess && run(6)) e = gla::launch_bwd_dv(s, dO, log_beta, dS_T, dv, dS0, w, hs);
  if (e == hipSuccess && run(7) && dlog_beta)
    e = gla::launch_beta_grad(s, o, dO, v, dv, dlog_beta, w, hs);
  return hip_status(e);
}

GLA_EXPORT gla_status gla_recurrent_fwd(const gla_problem *prob, const void *q, const void *k,
                                        const void *v, const void *log_alpha, const float *S0,
                                        void *o, float *S_T, void *stream) {
  return recurrent_fwd(prob, q, k, v, log_alpha, nullptr, S0, o, S_T, stream);
}

GLA_EXPORT gla_status gla_recurrent_fwd_general(const gla_problem *prob, const void *q, const void *k,
                                                const void *v, const void *log_alpha, const void *log_beta,
                                                const float *S0, void *o, float *S_T, void *stream) {
  return recurrent_fwd(prob, q, k, v, log_alpha, log_beta, S0, o, S_T, stream);
}

// ---------------------------------------------------------------- output side

namespace {

// The output side uses B, H, T, dv and io of the problem.
gla_status og_check(const gla_problem *p, float eps) {
  if (!p) return GLA_ERR_NULL;
  if (p->io != GLA_F32 && p->io != GLA_BF16) return GLA_ERR_DTYPE;
  if (p->B < 0 || p->H < 0 || p->T < 0 || p->dv <= 0) return GLA_ERR_SHAPE;
  if (!(eps > 0.f && eps < 3.0e38f)) return GLA_ERR_SHAPE;
  if (p->dv % 16 != 0 || p->dv > 1024) return GLA_ERR_UNSUPPORTED;
  const int64_t rows = (int64_t)p->B * p->H * p->T;
  if (rows >= (int64_t)1 << 31 || (int64_t)p->B * p->H > (1 << 24)) return GLA_ERR_UNSUPPORTED;
  return GLA_OK;
}

}  // namespace

GLA_EXPORT size_t gla_output_gate_workspace_bytes(const gla_problem *prob) {
  if (og_check(prob, 1.f) != GLA_OK) return 0;
  return gla::outgate_partial_bytes(prob->B, prob->H, prob->T, prob->dv);
}

GLA_EXPORT gla_status gla_output_gate_fwd(const gla_problem *prob, const void *o, const void *g,
                                          const float *ln_w, const float *ln_b, float eps, void *y,
                                          float *stats, void *stream) {
  gla_status st = og_check(prob, eps);
  if (st != GLA_OK) return st;
  const int64_t rows = (int64_t)prob->B * prob->H * prob->T;
  if (rows == 0) return GLA_OK;
  if (!o || !g || !y) return GLA_ERR_NULL;
  const int io = prob->io == GLA_BF16 ? gla::IO_BF16 : gla::IO_F32;
  return hip_status(gla::launch_outgate_fwd(prob->B, prob->H, prob->T, prob->dv, io, o, g, ln_w, ln_b, eps, y,
                                            stats, (hipStream_t)stream));
}

GLA_EXPORT gla_status gla_output_gate_bwd(const gla_problem *prob, const void *o, const void *g,
                                          const float *ln_w, const float *ln_b, float eps, const void *dy,
                                          void *d_o, void *dg, float *dln_w, float *dln_b, void *workspace,
                                          size_t workspace_bytes, void *stream) {
  gla_status st = og_check(prob, eps);
  if (st != GLA_OK) return st;
  const int64_t rows = (int64_t)prob->B * prob->H * prob->T;
  const bool affine = dln_w || dln_b;
  if (rows > 0 && (!o || !g || !dy || !d_o || !dg)) return GLA_ERR_NULL;
  if (rows == 0 && (!affine || prob->H == 0)) return GLA_OK;  // (no rows: zero affine gradients below)
  const size_t need = affine ? gla::outgate_partial_bytes(prob->B, prob->H, prob->T, prob->dv) : 0;
  if (affine && need > 0 && (!workspace || workspace_bytes < need)) return GLA_ERR_WORKSPACE;
  const int io = prob->io == GLA_BF16 ? gla::IO_BF16 : gla::IO_F32;
  return hip_status(gla::launch_outgate_bwd(prob->B, prob->H, prob->T, prob->dv, io, o, g, ln_w, ln_b, eps, dy,
                                            d_o, dg, dln_w, dln_b, (float *)workspace, (hipStream_t)stream));
}
