// Decoder context: buffers, prefill and the SJD-PAC step (window forward,
// verification, KV commit), all enqueued on the caller's stream. The host
// never reads device state during a step except to keep a bound on the
// cache fill (one 4-byte copy per step into pinned memory, polled without
// blocking).
#include <hip/hip_runtime.h>

#include <array>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <utility>
#include <vector>

#include "forward.h"
#include "sjd.h"
#include "step.h"
#include "verify.h"

namespace {

constexpr int kRing = 8;

struct Ctx {
  sjd_config c{};
  int cap = 0;      // KV rows
  int cap_pad = 0;  // row stride of the caches (multiple of the attention chunk)
  int Mpad = 64;  // activation rows (window rows: one stream of <= 64, or up to four streams of 32)
  static constexpr int kPrefillRows = 64;  // prefill windows (one stream)
  // library-owned weights: embedding and norm gains as bf16 rows, matrices
  // in the GEMM tile layout; lw[l] = {attn_norm, wqkv, -, -, wo, ffn_norm, wgu, -, wd}
  const uint16_t* embed = nullptr;
  const uint16_t* fnorm = nullptr;
  const uint16_t* head = nullptr;
  std::vector<std::array<const uint16_t*, 9>> lw;
  int ld_d = 0, ld_q = 0, ld_f = 0;  // padded row strides of the activation planes
  std::vector<void*> owned;
  // activations entering MFMAs are hi / lo bf16 plane pairs
  float* x = nullptr;
  uint16_t *xn = nullptr, *xn_lo = nullptr;
  float* qkv = nullptr;
  uint16_t *q = nullptr, *q_lo = nullptr;
  uint16_t *att = nullptr, *att_lo = nullptr;
  uint16_t *hbuf = nullptr, *hbuf_lo = nullptr;
  uint16_t *kc = nullptr, *kc_lo = nullptr;
  uint16_t *vt = nullptr, *vt_lo = nullptr;
  // streams: one per image of a batch (up to four), two per image for a
  // guided context (text prompt + unconditional stream; up to two images);
  // stream z's caches start z * kv_elems elements into kc.. (an
  // unconditional stream's positions are its text stream's plus the image's
  // delta = n_uncond - n_prompt, kept in the image's device state)
  bool guided = false;
  int B = 1;         // images per step
  int nstreams = 1;
  size_t kv_elems = 0;
  int delta[sjd::kMaxStreams] = {0, 0, 0, 0};  // per image (host copy, for the cache-fill bound)
  float2* rope = nullptr;
  float* logits[2] = {nullptr, nullptr};
  // target-row statistics of the step that wrote logits[i] ([B][L]); the
  // next step's draft rows reuse them instead of selecting again
  sjd::RowStatsCache* stats[2] = {nullptr, nullptr};
  float* attn_o = nullptr;
  float* attn_ml = nullptr;
  int nsplit_max = 0;
  float* rpart = nullptr;  // split-K partial planes of the O / down projections
  float* gup = nullptr;    // split-K partial planes of the gate / up projection [S_gu][Mpad][2F]
  float* ss = nullptr;     // RMSNorm chunk sums of squares [Mpad][norm_chunks(d)]
  sjd::DevState* st = nullptr;
  sjd::Window* win = nullptr;
  int32_t* rec = nullptr;
  int32_t* nonfinite = nullptr;  // SJD_CHECK_FINITE: count of NaN / +inf logits found
  // GEMM plan per projection (QKV, O, gate|up, down): split count and column
  // blocks per workgroup, for windows of <= 32 rows [0] and of more [1]
  // (two streams, L > 32, prefill windows); the LM head runs wide, unsplit
  struct Plan {
    int S = 1, wide = 0;
  };
  Plan plan[2][4];
  // windows of more than 64 rows (three or four streams): the 64-row plan
  // with each projection's splits cut to fit one workgroup per compute unit
  // (a 96- or 128-row workgroup holds three or four accumulator tiles and
  // only one fits a compute unit; a larger grid runs in two rounds)
  Plan plan_wide[4];
  long long steps = 0;
  unsigned prefilled = 0;  // bit b: image b prefilled
  // attention workgroups per key / value head (its grouped query heads split
  // over them)
  int qparts = 1;
  // the step's window forward (window build + ~10 kernels per layer + head),
  // captured once per logits buffer on cap_stream and replayed on the
  // caller's stream: its kernels and arguments never change for a context
  bool use_graph = true;
  hipStream_t cap_stream = nullptr;
  hipGraphExec_t fwd_exec[2] = {nullptr, nullptr};
  // cache-fill bound, per image: cached rows after step ev_step[i] are
  // written by the step's last kernel into h_n[i * B + b] (pinned host ring)
  int32_t* h_n = nullptr;
  int32_t* h_n_dev = nullptr;  // its device-side address
  hipEvent_t ev[kRing];
  long long ev_step[kRing];
  long long known_step[sjd::kMaxStreams] = {-1, -1, -1, -1};  // step after which known_n holds
  long long img_step0[sjd::kMaxStreams] = {0, 0, 0, 0};      // first step of the image's current generation
  int known_n[sjd::kMaxStreams] = {0, 0, 0, 0};
  int n_events = 0;
};

template <class T>
int dalloc(Ctx& x, T** p, size_t count) {
  void* q = nullptr;
  if (hipMalloc(&q, count * sizeof(T) > 0 ? count * sizeof(T) : 16) != hipSuccess) return SJD_ENOMEM;
  x.owned.push_back(q);
  *p = (T*)q;
  return SJD_OK;
}

// rows of a step's logits buffer: image b's rows at [32 b, 32 b + L) (a
// guided head writes each image's guided rows there)
int logit_rows(const Ctx& x) { return 32 * (x.B - 1) + x.c.L; }

int check_config(const sjd_config* c) {
  if (!c) return SJD_EINVAL;
  if (c->n_layers < 1 || c->d_model < 64 || c->d_model % 64 || c->n_heads < 1 || c->n_kv_heads < 1 ||
      c->n_heads % c->n_kv_heads)
    return SJD_EINVAL;
  if (c->head_dim != 64 && c->head_dim != 128) return SJD_ENOTSUP;
  if ((c->n_heads * c->head_dim) % 64 || c->ffn_dim < 64 || c->ffn_dim % 64) return SJD_EINVAL;
  if (c->vocab_size < 1 || c->V < 32 || c->V % 32 || c->vis_lo < 0 || c->vis_lo + c->V > c->vocab_size)
    return SJD_EINVAL;
  if (c->L < 1 || c->L > 64 || c->K < 1 || c->K > 8 || c->D < 0 || (long)c->K * c->D > c->L) return SJD_EINVAL;
  if (c->V > 65536) return SJD_ENOTSUP;
  if (c->max_seq < c->L + 2) return SJD_EINVAL;
  if (c->flags & ~(SJD_AC | SJD_PD | SJD_EAGER | SJD_NO_TUNE | SJD_TUNE | SJD_CHECK_FINITE)) return SJD_EINVAL;
  if (!(c->rms_eps > 0.0f) || !(c->rope_theta > 0.0f)) return SJD_EINVAL;
  if (!std::isfinite(c->cfg_w)) return SJD_EINVAL;
  if (c->batch < 0) return SJD_EINVAL;
  const int B = c->batch > 1 ? c->batch : 1;
  const int nz = B * (c->cfg_w != 0.0f ? 2 : 1);
  if (nz > sjd::kMaxStreams) return SJD_ENOTSUP;  // streams of 32 rows in 128
  if (nz > 1 && c->L > 32) return SJD_ENOTSUP;
  return SJD_OK;
}

#define TRY(e)                          \
  do {                                  \
    int _rc = (e);                      \
    if (_rc != SJD_OK) return _rc;      \
  } while (0)
#define HIPTRY(e)                                \
  do {                                           \
    if ((e) != hipSuccess) return SJD_EHIP;      \
  } while (0)

enum { kProjQkv = 0, kProjO = 1, kProjGu = 2, kProjDown = 3 };

// Window forward of M rows: two streams (sm.mode != kStreamsOne, see
// Streams), or one stream on the caches of stream `cache` (a prefill).
int forward(Ctx& x, int M, const int32_t* n_dev, int n_host, float* logits, const sjd::Streams& sm, int cache,
            hipStream_t s) {
  const sjd_config& c = x.c;
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  const int Nq = H * hd, Nkv = Hkv * hd, Nqkv = Nq + 2 * Nkv;
  HIPTRY(sjd::launch_embed(x.embed, x.win, M, d, c.vocab_size, c.vis_lo, x.x, s));
  const size_t qplane = (size_t)x.Mpad * Nqkv, rplane = (size_t)x.Mpad * d, guplane = (size_t)x.Mpad * 2 * F;
  int pend = 0;  // partial planes of the last residual projection not yet added into x
  const Ctx::Plan* P = M > 64 ? x.plan_wide : x.plan[M > 32 ? 1 : 0];
  sjd::GemmArgs normed{};  // GEMM arguments that apply the RMSNorm row scale
  normed.ss = x.ss;
  normed.ss_n = sjd::norm_chunks(d);
  normed.inv_d = 1.0f / (float)d;
  normed.eps = c.rms_eps;
  for (int l = 0; l < c.n_layers; ++l) {
    const auto& w = x.lw[l];
    const size_t lofs = (size_t)l * Hkv * x.cap_pad * hd + (size_t)cache * x.kv_elems;
    sjd::KvPlanes kv{x.q, x.q_lo, x.kc + lofs, x.kc_lo + lofs, x.vt + lofs, x.vt_lo + lofs, x.kv_elems};
    HIPTRY(sjd::launch_resid_norm(x.x, x.rpart, pend, rplane, w[0], M, d, x.xn, x.xn_lo, x.ld_d, x.ss, s));
    sjd::GemmArgs g = normed;
    g.A = x.xn; g.A_lo = x.xn_lo; g.lda = x.ld_d; g.M = M; g.W = w[1]; g.N = Nqkv; g.K = d; g.S = P[kProjQkv].S;
    g.wide = P[kProjQkv].wide; g.out = x.qkv; g.plane = qplane; g.ldo = Nqkv;
    HIPTRY(sjd::launch_gemm(g, s));
    HIPTRY(sjd::launch_rope_kv(x.qkv, P[kProjQkv].S, qplane, x.win, n_dev, n_host, M, H, Hkv, hd, x.rope, kv, x.cap_pad,
                               sm, s));
    sjd::AttnArgs a{};
    a.q = x.q; a.q_lo = x.q_lo; a.kc = kv.kc; a.kc_lo = kv.kc_lo; a.vt = kv.vt; a.vt_lo = kv.vt_lo; a.win = x.win;
    a.sstride = kv.sstride; a.st = sm;
    a.n_dev = n_dev; a.n_host = n_host; a.M = M; a.H = H; a.Hkv = Hkv; a.cap = x.cap_pad;
    a.scale = (float)(1.4426950408889634 / std::sqrt((double)hd));
    a.ws_o = x.attn_o; a.ws_ml = x.attn_ml; a.nsplit_max = x.nsplit_max; a.out = x.att; a.out_lo = x.att_lo;
    a.ldo = x.ld_q; a.qparts = x.qparts;
    HIPTRY(sjd::launch_attention(a, hd, s));
    g = sjd::GemmArgs{};
    g.A = x.att; g.A_lo = x.att_lo; g.lda = x.ld_q; g.M = M; g.W = w[4]; g.N = d; g.K = Nq; g.S = P[kProjO].S;
    g.wide = P[kProjO].wide; g.out = x.rpart; g.plane = rplane; g.ldo = d;
    HIPTRY(sjd::launch_gemm(g, s));
    HIPTRY(sjd::launch_resid_norm(x.x, x.rpart, P[kProjO].S, rplane, w[5], M, d, x.xn, x.xn_lo, x.ld_d, x.ss, s));
    g = normed;
    g.A = x.xn; g.A_lo = x.xn_lo; g.lda = x.ld_d; g.M = M; g.W = w[6]; g.N = 2 * F; g.K = d; g.S = P[kProjGu].S;
    g.wide = P[kProjGu].wide; g.out = x.gup; g.plane = guplane; g.ldo = 2 * F;
    HIPTRY(sjd::launch_gemm(g, s));
    HIPTRY(sjd::launch_swiglu(x.gup, P[kProjGu].S, guplane, M, F, x.hbuf, x.hbuf_lo, x.ld_f, s));
    g = sjd::GemmArgs{};
    g.A = x.hbuf; g.A_lo = x.hbuf_lo; g.lda = x.ld_f; g.M = M; g.W = w[8]; g.N = d; g.K = F; g.S = P[kProjDown].S;
    g.wide = P[kProjDown].wide; g.out = x.rpart; g.plane = rplane; g.ldo = d;
    HIPTRY(sjd::launch_gemm(g, s));
    pend = P[kProjDown].S;
  }
  if (logits) {
    HIPTRY(sjd::launch_resid_norm(x.x, x.rpart, pend, rplane, x.fnorm, M, d, x.xn, x.xn_lo, x.ld_d, x.ss, s));
    sjd::GemmArgs g = normed;
    g.A = x.xn; g.A_lo = x.xn_lo; g.lda = x.ld_d; g.M = M; g.W = x.head; g.N = c.V; g.K = d; g.S = 1;
    g.wide = 1;  // measured faster at 32 and 64 rows
    g.out = logits; g.plane = 0; g.ldo = c.V;
    if (sm.mode == sjd::kStreamsMulti && sm.guided) {  // rows [32 b, 32 b + L): image b's guided logits
      g.cfg_rows = sm.L;
      g.cfg_w = c.cfg_w;
    }
    HIPTRY(sjd::launch_gemm(g, s));
  }
  return SJD_OK;
}

// ---- split-K plan
// How many workgroups share a projection's K range decides both the GEMM's
// time and how many partial planes its consumer (RoPE, residual + RMSNorm,
// SwiGLU) sums; the interaction is not smooth (measured on the 7B shape, the
// step is 3% faster with the timed plan than with the closed form). The
// split count also sets the summation order, so the plan must not depend on
// timing by default: a context takes the plan recorded for its shape (the
// choice of the timed search below on MI355X, for the shapes listed), else
// the closed form. With SJD_TUNE the first context of a process that meets a
// projection shape times every candidate pair (GEMM + consumer) on its own
// weights and keeps the fastest for the process: every context of the
// process uses the same plan, so their arithmetic agrees.
struct RecordedPlan {
  int kind, N, K, cls, S, wide;
};
const RecordedPlan kRecordedPlans[] = {
    // {projection (0 QKV, 1 O, 2 gate|up, 3 down), N, K, row class (0: windows
    //  of <= 32 rows, 1: more), splits, 8 column blocks per workgroup}
    // 7B shape (d 4096, 32 x 128 heads, FFN 11008)
    {0, 12288, 4096, 0, 5, 1}, {1, 4096, 4096, 0, 8, 0}, {2, 22016, 4096, 0, 2, 1}, {3, 4096, 11008, 0, 8, 0},
    {0, 12288, 4096, 1, 5, 1}, {1, 4096, 4096, 1, 8, 0}, {2, 22016, 4096, 1, 2, 1}, {3, 4096, 11008, 1, 15, 1},
    // 8B GQA shape (d 4096, 32 / 8 x 128 heads, FFN 14336); its O projection is the 7B one
    {0, 6144, 4096, 0, 5, 0}, {2, 28672, 4096, 0, 2, 1}, {3, 4096, 14336, 0, 8, 0},
    {0, 6144, 4096, 1, 5, 0}, {2, 28672, 4096, 1, 2, 1}, {3, 4096, 14336, 1, 16, 1},
    // mid shape (d 1024, 16 x 64 heads, FFN 2816)
    {0, 3072, 1024, 0, 8, 0}, {1, 1024, 1024, 0, 8, 0}, {2, 5632, 1024, 0, 5, 0}, {3, 1024, 2816, 0, 22, 0},
    {0, 3072, 1024, 1, 8, 0}, {2, 5632, 1024, 1, 5, 0},
};

bool recorded_plan(int kind, int N, int K, int cls, Ctx::Plan* out) {
  for (const RecordedPlan& r : kRecordedPlans)
    if (r.kind == kind && r.N == N && r.K == K && r.cls == cls) {
      *out = Ctx::Plan{r.S, r.wide};
      return true;
    }
  return false;
}

std::mutex g_plan_mu;
// (projection, N, K, row class) -> plan
std::map<std::tuple<int, int, int, int>, Ctx::Plan> g_plan;

// candidate plans: 4 and 8 column blocks per workgroup, half a workgroup to
// three workgroups per compute unit (a grid just short of one per unit
// leaves a few idle but none doubled up: the 7B QKV projection ran fastest
// at 5 splits of 48 eight-block groups, 240 workgroups; fewer splits mean
// fewer partial planes for the consumer to sum, which can outweigh a
// slower GEMM), at least two k-steps per workgroup, plus the closed-form
// choice
std::vector<Ctx::Plan> plan_candidates(int N, int K, int ncu, Ctx::Plan fallback) {
  const int T = K / 64;
  std::vector<Ctx::Plan> out;
  for (int wide = 0; wide < 2; ++wide) {
    const int nw = wide ? 8 : 4;
    const int groups = (N / 32 + nw - 1) / nw;
    for (int S = 1; S <= sjd::kGemmMaxSplits; ++S) {
      if (S > 1 && T / S < 2) break;
      const long wg = (long)groups * S;
      if (2 * wg >= (long)ncu && wg <= 3L * ncu) out.push_back(Ctx::Plan{S, wide});
    }
  }
  bool has = false;
  for (const Ctx::Plan& p : out) has |= p.S == fallback.S && p.wide == fallback.wide;
  if (!has) out.push_back(fallback);
  return out;
}

// Times GEMM + consumer per candidate (M rows, current buffer contents) and
// returns the chosen plan (see below; S < 1: error). Repetition r runs layer
// r's weights (mod the layer count): the projections of the large models
// fit in the 256 MB last-level cache one layer at a time, and a plan timed
// on cache-resident weights is not the one that streams fastest from HBM.
Ctx::Plan tune_projection(Ctx& x, int proj, const std::vector<Ctx::Plan>& cand, Ctx::Plan closed, int M,
                          hipStream_t s) {
  const sjd_config& c = x.c;
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  const int Nq = H * hd, Nkv = Hkv * hd, Nqkv = Nq + 2 * Nkv;
  const Ctx::Plan fail{0, 0};
  const size_t qplane = (size_t)x.Mpad * Nqkv, rplane = (size_t)x.Mpad * d, guplane = (size_t)x.Mpad * 2 * F;
  const sjd::Streams one{sjd::kStreamsOne, 0, 0, 0, nullptr};
  auto pair = [&](const Ctx::Plan& pl, int rep) -> hipError_t {
    const auto& w = x.lw[rep % c.n_layers];
    const int S = pl.S;
    sjd::GemmArgs g{};
    g.M = M; g.S = S; g.wide = pl.wide;
    if (proj == kProjQkv || proj == kProjGu) {
      g.ss = x.ss; g.ss_n = sjd::norm_chunks(d); g.inv_d = 1.0f / (float)d; g.eps = c.rms_eps;
      g.A = x.xn; g.A_lo = x.xn_lo; g.lda = x.ld_d; g.K = d;
    }
    hipError_t e;
    switch (proj) {
      case kProjQkv: {
        g.W = w[1]; g.N = Nqkv; g.out = x.qkv; g.plane = qplane; g.ldo = Nqkv;
        if ((e = sjd::launch_gemm(g, s)) != hipSuccess) return e;
        const sjd::KvPlanes kv{x.q, x.q_lo, x.kc, x.kc_lo, x.vt, x.vt_lo, x.kv_elems};
        return sjd::launch_rope_kv(x.qkv, S, qplane, x.win, nullptr, 0, M, H, Hkv, hd, x.rope, kv, x.cap_pad, one, s);
      }
      case kProjO:
        g.A = x.att; g.A_lo = x.att_lo; g.lda = x.ld_q; g.W = w[4]; g.N = d; g.K = Nq;
        g.out = x.rpart; g.plane = rplane; g.ldo = d;
        if ((e = sjd::launch_gemm(g, s)) != hipSuccess) return e;
        return sjd::launch_resid_norm(x.x, x.rpart, S, rplane, w[5], M, d, x.xn, x.xn_lo, x.ld_d, x.ss, s);
      case kProjGu:
        g.W = w[6]; g.N = 2 * F; g.out = x.gup; g.plane = guplane; g.ldo = 2 * F;
        if ((e = sjd::launch_gemm(g, s)) != hipSuccess) return e;
        return sjd::launch_swiglu(x.gup, S, guplane, M, F, x.hbuf, x.hbuf_lo, x.ld_f, s);
      default:
        g.A = x.hbuf; g.A_lo = x.hbuf_lo; g.lda = x.ld_f; g.W = w[8]; g.N = d; g.K = F;
        g.out = x.rpart; g.plane = rplane; g.ldo = d;
        if ((e = sjd::launch_gemm(g, s)) != hipSuccess) return e;
        return sjd::launch_resid_norm(x.x, x.rpart, S, rplane, w[0], M, d, x.xn, x.xn_lo, x.ld_d, x.ss, s);
    }
  };
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    return fail;
  }
  // two interleaved rounds over the candidates; each keeps its faster round
  constexpr int kReps = 10, kRounds = 2;
  std::vector<float> t(cand.size(), 0.0f);
  bool ok = true;
  for (int round = 0; round < kRounds && ok; ++round)
    for (size_t i = 0; i < cand.size() && ok; ++i) {
      const Ctx::Plan pl = cand[i];
      for (int r = 0; r < 2 && ok; ++r) ok = pair(pl, kReps + r) == hipSuccess;
      ok = ok && hipEventRecord(e0, s) == hipSuccess;
      for (int r = 0; r < kReps && ok; ++r) ok = pair(pl, r) == hipSuccess;
      ok = ok && hipEventRecord(e1, s) == hipSuccess && hipEventSynchronize(e1) == hipSuccess;
      float ms = 0.0f;
      ok = ok && hipEventElapsedTime(&ms, e0, e1) == hipSuccess;
      const float us = ms * 1e3f / kReps;
      if (round == 0 || us < t[i]) t[i] = us;
    }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (!ok) return fail;
  // the closed-form choice unless a candidate beats it by more than 3%
  // (then the fastest): near-ties keep the same plan however noisy the
  // timing (another process, a profiler attached)
  size_t ref = 0;
  for (size_t i = 0; i < t.size(); ++i)
    if (cand[i].S == closed.S && cand[i].wide == closed.wide) ref = i;
  size_t pick = ref;
  for (size_t i = 0; i < t.size(); ++i)
    if (t[i] < t[ref] * 0.97f && t[i] < t[pick]) pick = i;
  if (std::getenv("SJD_LOG_PLAN"))
    for (size_t i = 0; i < t.size(); ++i)
      std::fprintf(stderr, "[sjd] plan: projection %d, %d rows: %d splits x %d blocks: %.2f us%s\n", proj, M,
                   cand[i].S, cand[i].wide ? 8 : 4, t[i], i == pick ? " <- chosen" : "");
  return cand[pick];
}

// Refreshes the cache-fill bound of every image from completed steps;
// blocks only when the bound says the next window might not fit.
int cache_check(Ctx& x) {
  for (int b = 0; b < x.B; ++b) {
    const int ahead = x.delta[b] > 0 ? x.delta[b] : 0;  // an unconditional stream runs ahead by delta
    auto refresh = [&](bool wait) -> int {
      for (int i = 0; i < kRing; ++i) {
        if (x.ev_step[i] <= x.known_step[b] || x.ev_step[i] < x.img_step0[b]) continue;
        if (wait && x.ev_step[i] == x.steps - 1) HIPTRY(hipEventSynchronize(x.ev[i]));
        if (hipEventQuery(x.ev[i]) == hipSuccess) {
          x.known_step[b] = x.ev_step[i];
          x.known_n[b] = x.h_n[i * x.B + b];
        }
      }
      return SJD_OK;
    };
    TRY(refresh(false));
    long long pending = x.steps - 1 - x.known_step[b];
    if ((long long)x.known_n[b] + ahead + pending * x.c.L + x.c.L <= x.cap) continue;
    TRY(refresh(true));  // wait for the newest step and use its exact value
    pending = x.steps - 1 - x.known_step[b];
    if ((long long)x.known_n[b] + ahead + pending * x.c.L + x.c.L > x.cap) return SJD_ESTATE;
  }
  return SJD_OK;
}

}  // namespace

struct sjd_ctx {
  Ctx x;
};

extern "C" int sjd_init(const sjd_config* cfg, const sjd_weights* w, void* stream, sjd_ctx** out) {
  if (!out) return SJD_EINVAL;
  *out = nullptr;
  TRY(check_config(cfg));
  if (!w || !w->d_embed || !w->h_layer || !w->d_final_norm || !w->d_lm_head) return SJD_EINVAL;
  for (int i = 0; i < 9 * cfg->n_layers; ++i)
    if (!w->h_layer[i]) return SJD_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  sjd_ctx* h = new sjd_ctx();
  Ctx& x = h->x;
  x.c = *cfg;
  const sjd_config& c = x.c;
  x.guided = c.cfg_w != 0.0f;
  x.use_graph = !(c.flags & SJD_EAGER);
  x.B = c.batch > 1 ? c.batch : 1;
  x.nstreams = x.B * (x.guided ? 2 : 1);
  x.Mpad = x.nstreams > 2 ? 32 * x.nstreams : 64;
  auto fail = [&](int rc) {
    sjd_destroy(h);
    return rc;
  };
  const int d = c.d_model, H = c.n_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.ffn_dim;
  const int Nq = H * hd, Nkv = Hkv * hd;
  x.cap = c.max_seq;
  x.cap_pad = ((c.max_seq + sjd::kAttnChunk - 1) / sjd::kAttnChunk) * sjd::kAttnChunk;
  x.nsplit_max = x.cap_pad / sjd::kAttnChunk;

  // weights: copied into library memory; matrices repacked into the GEMM
  // tile layout (bf16), fp32 inputs rounded to nearest even
  const int f32 = c.weights_f32 ? 1 : 0;
  auto copy_rows = [&](const void* p, size_t count, const uint16_t** dst) -> int {
    uint16_t* b = nullptr;
    int rc = dalloc(x, &b, count);
    if (rc != SJD_OK) return rc;
    if (f32) {
      if (sjd::launch_f32_to_bf16((const float*)p, b, count, s) != hipSuccess) return SJD_EHIP;
    } else if (hipMemcpyAsync(b, p, count * 2, hipMemcpyDeviceToDevice, s) != hipSuccess) {
      return SJD_EHIP;
    }
    *dst = b;
    return SJD_OK;
  };
  // rows [row0, row0 + N) of src ([*][K]) as row blocks [nb0, nb0 + N/32) of
  // a tiled matrix of Ntot rows at dst
  auto tile = [&](const void* p, size_t row0, int N, int K, uint16_t* dst, int Ntot, int nb0) -> int {
    return sjd::launch_tile_weights(p, f32, row0, N, K, dst, Ntot / 32, nb0, s) == hipSuccess ? SJD_OK
                                                                                             : SJD_EHIP;
  };
  int rc = copy_rows(w->d_embed, (size_t)c.vocab_size * d, &x.embed);
  if (rc == SJD_OK) rc = copy_rows(w->d_final_norm, d, &x.fnorm);
  if (rc == SJD_OK) {
    uint16_t* hp = nullptr;
    rc = dalloc(x, &hp, (size_t)c.V * d);
    if (rc == SJD_OK) rc = tile(w->d_lm_head, (size_t)c.vis_lo, c.V, d, hp, c.V, 0);
    x.head = hp;
  }
  x.lw.resize(c.n_layers);
  for (int l = 0; l < c.n_layers && rc == SJD_OK; ++l) {
    const void* const* lp = w->h_layer + 9 * l;
    auto& o = x.lw[l];
    rc = copy_rows(lp[0], d, &o[0]);
    if (rc == SJD_OK) rc = copy_rows(lp[5], d, &o[5]);
    uint16_t *qkv = nullptr, *wo = nullptr, *wgu = nullptr, *wd = nullptr;
    const size_t tq = (size_t)Nq * d, tkv = (size_t)Nkv * d;
    if (rc == SJD_OK) rc = dalloc(x, &qkv, tq + 2 * tkv);
    const int Nqkv = Nq + 2 * Nkv;
    if (rc == SJD_OK) rc = tile(lp[1], 0, Nq, d, qkv, Nqkv, 0);
    if (rc == SJD_OK) rc = tile(lp[2], 0, Nkv, d, qkv, Nqkv, Nq / 32);
    if (rc == SJD_OK) rc = tile(lp[3], 0, Nkv, d, qkv, Nqkv, (Nq + Nkv) / 32);
    if (rc == SJD_OK) rc = dalloc(x, &wo, (size_t)d * Nq);
    if (rc == SJD_OK) rc = tile(lp[4], 0, d, Nq, wo, d, 0);
    if (rc == SJD_OK) rc = dalloc(x, &wgu, (size_t)2 * F * d);
    if (rc == SJD_OK) rc = tile(lp[6], 0, F, d, wgu, 2 * F, 0);
    if (rc == SJD_OK) rc = tile(lp[7], 0, F, d, wgu, 2 * F, F / 32);
    if (rc == SJD_OK) rc = dalloc(x, &wd, (size_t)d * F);
    if (rc == SJD_OK) rc = tile(lp[8], 0, d, F, wd, d, 0);
    o[1] = qkv; o[2] = nullptr; o[3] = nullptr; o[4] = wo; o[6] = wgu; o[7] = nullptr; o[8] = wd;
  }
  if (rc != SJD_OK) return fail(rc);
  // the caller may release its weights once sjd_init returns
  if (hipStreamSynchronize(s) != hipSuccess) return fail(SJD_EHIP);

  // work buffers
  const int Mp = x.Mpad;
  x.kv_elems = (size_t)c.n_layers * Hkv * x.cap_pad * hd;
  const size_t kv = x.kv_elems * x.nstreams;  // every stream's caches
  // activation rows padded by 64 elements so that the 32 rows a wave reads per
  // k-step spread over memory channels
  x.ld_d = d + 64;
  x.ld_q = Nq + 64;
  x.ld_f = F + 64;
  const size_t xnsz = (size_t)Mp * x.ld_d;
  if ((rc = dalloc(x, &x.x, (size_t)Mp * d)) || (rc = dalloc(x, &x.xn, xnsz)) || (rc = dalloc(x, &x.xn_lo, xnsz)) ||
      (rc = dalloc(x, &x.q, (size_t)Mp * Nq)) ||
      (rc = dalloc(x, &x.q_lo, (size_t)Mp * Nq)) || (rc = dalloc(x, &x.att, (size_t)Mp * x.ld_q)) ||
      (rc = dalloc(x, &x.att_lo, (size_t)Mp * x.ld_q)) || (rc = dalloc(x, &x.hbuf, (size_t)Mp * x.ld_f)) ||
      (rc = dalloc(x, &x.hbuf_lo, (size_t)Mp * x.ld_f)) || (rc = dalloc(x, &x.kc, kv)) || (rc = dalloc(x, &x.kc_lo, kv)) ||
      (rc = dalloc(x, &x.vt, kv)) || (rc = dalloc(x, &x.vt_lo, kv)) ||
      (rc = dalloc(x, &x.rope, (size_t)x.cap_pad * (hd / 2))) ||
      (rc = dalloc(x, &x.logits[0], (size_t)logit_rows(x) * c.V)) ||
      (rc = dalloc(x, &x.logits[1], (size_t)logit_rows(x) * c.V)) ||
      (rc = dalloc(x, &x.stats[0], (size_t)x.B * c.L)) || (rc = dalloc(x, &x.stats[1], (size_t)x.B * c.L)) ||
      (rc = dalloc(x, &x.attn_o, (size_t)H * x.nsplit_max * sjd::kWinRows * hd)) ||
      (rc = dalloc(x, &x.attn_ml, (size_t)H * x.nsplit_max * sjd::kWinRows * 2)) || (rc = dalloc(x, &x.st, x.B)) ||
      (rc = dalloc(x, &x.win, 1)) || (rc = dalloc(x, &x.rec, (size_t)x.B * c.L * sjd::kRecInts)) ||
      (rc = dalloc(x, &x.nonfinite, 16)))
    return fail(rc);
  // split-K plan: the closed form aims for two to three workgroups per
  // compute unit; unless SJD_NO_TUNE, the process-wide tuned plan replaces it
  // (tuned below, by the first context that meets a shape)
  int ncu = 256;
  {
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
      ncu = prop.multiProcessorCount;
  }
  const int target = 5 * ncu / 2;
  // grouped-query attention: one attention workgroup per query head by
  // default (the parts of a key / value head share an XCD and its L2, so the
  // head's tiles still come from HBM once); SJD_QPARTS=p takes G / p query
  // heads per workgroup (p must divide G)
  {
    const int G = H / Hkv;
    const char* e = std::getenv("SJD_QPARTS");
    int qp = G;
    if (e && *e) {
      char* end = nullptr;
      const long v = std::strtol(e, &end, 10);
      if (*end != '\0' || v < 1 || G % v) return fail(SJD_EINVAL);
      qp = (int)v;
    }
    x.qparts = qp;
  }
  const int Nqkv = Nq + 2 * Nkv;
  // one plan per projection and row class (windows of <= 32 rows; of more:
  // timed only for contexts whose steps run them, else the closed form, which
  // serves their 64-row prefill windows)
  const int kind_N[4] = {Nqkv, d, 2 * F, d}, kind_K[4] = {d, Nq, d, F};
  const bool step64 = x.nstreams > 1 || c.L > 32;
  struct Proj { int kind, N, K, cls; Ctx::Plan closed; std::vector<Ctx::Plan> cand; bool tune; };
  std::vector<Proj> projs;
  for (int cls = 0; cls < 2; ++cls)
    for (int k = 0; k < 4; ++k) {
      Proj p{k, kind_N[k], kind_K[k], cls, Ctx::Plan{}, {}, false};
      p.closed = Ctx::Plan{sjd::gemm_splits(p.N, p.K, target, cls == 1), cls};
      projs.push_back(p);
    }
  // SJD_SPLITS="qkv,o,gu,down" pins the plan of windows of <= 32 rows (e.g.
  // to profile the plan a run without the profiler chose); an entry "S:8"
  // runs 8 column blocks per workgroup, "S" or "S:4" four; unset or empty:
  // no pin
  Ctx::Plan pin[4];
  bool pinned = false;
  const char* env = std::getenv("SJD_SPLITS");
  if (env && *env) {
    const char* q = env;
    for (int i = 0; i < 4; ++i) {
      char* end = nullptr;
      const long v = std::strtol(q, &end, 10);
      if (end == q || v < 1 || v > sjd::kGemmMaxSplits) return fail(SJD_EINVAL);
      long wv = 4;
      if (*end == ':') {
        q = end + 1;
        wv = std::strtol(q, &end, 10);
        if (end == q || (wv != 4 && wv != 8)) return fail(SJD_EINVAL);
      }
      if (*end != (i < 3 ? ',' : '\0')) return fail(SJD_EINVAL);
      pin[i] = Ctx::Plan{(int)v, wv == 8 ? 1 : 0};
      q = end + 1;
    }
    pinned = true;
  }
  const bool tune = (c.flags & SJD_TUNE) && !(c.flags & SJD_NO_TUNE) && !pinned;
  const bool recorded = !(c.flags & (SJD_TUNE | SJD_NO_TUNE));
  int smax[4] = {1, 1, 1, 1};
  {
    std::lock_guard<std::mutex> lk(g_plan_mu);
    for (Proj& p : projs) {
      Ctx::Plan& dst = x.plan[p.cls][p.kind];
      dst = pinned && p.cls == 0 ? pin[p.kind] : p.closed;
      if (recorded && !(pinned && p.cls == 0)) recorded_plan(p.kind, p.N, p.K, p.cls, &dst);
      if (tune && (p.cls == 0 || step64)) {
        auto it = g_plan.find(std::make_tuple(p.kind, p.N, p.K, p.cls));
        if (it != g_plan.end()) {
          dst = it->second;
        } else {
          p.cand = plan_candidates(p.N, p.K, ncu, p.closed);
          p.tune = true;
        }
      }
      smax[p.kind] = dst.S > smax[p.kind] ? dst.S : smax[p.kind];
      for (const Ctx::Plan& q : p.cand) smax[p.kind] = q.S > smax[p.kind] ? q.S : smax[p.kind];
    }
  }
  const int sr = smax[1] > smax[3] ? smax[1] : smax[3];
  if ((rc = dalloc(x, &x.qkv, (size_t)smax[0] * Mp * Nqkv)) ||
      (rc = dalloc(x, &x.rpart, (size_t)sr * Mp * d)) ||
      (rc = dalloc(x, &x.gup, (size_t)smax[2] * Mp * 2 * F)) ||
      (rc = dalloc(x, &x.ss, (size_t)Mp * sjd::norm_chunks(d))))
    return fail(rc);
  // zero the caches (rows past the fill are read, masked, by the attention
  // tiles), the window and the activation planes (pad rows stay finite)
  bool ok0 = true;
  for (auto* st : x.stats) ok0 = ok0 && hipMemsetAsync(st, 0, sizeof(sjd::RowStatsCache) * x.B * c.L, s) == hipSuccess;
  void* zero[] = {x.kc, x.kc_lo, x.vt, x.vt_lo};
  bool ok = ok0 && hipMemsetAsync(x.st, 0, sizeof(sjd::DevState) * x.B, s) == hipSuccess;
  ok = ok && hipMemsetAsync(x.win, 0, sizeof(sjd::Window), s) == hipSuccess;
  ok = ok && hipMemsetAsync(x.x, 0, (size_t)Mp * d * sizeof(float), s) == hipSuccess;
  for (void* p : zero) ok = ok && hipMemsetAsync(p, 0, kv * 2, s) == hipSuccess;
  void* zero2[] = {x.xn, x.xn_lo};
  for (void* p : zero2) ok = ok && hipMemsetAsync(p, 0, xnsz * 2, s) == hipSuccess;
  void* zero3[] = {x.att, x.att_lo};
  for (void* p : zero3) ok = ok && hipMemsetAsync(p, 0, (size_t)Mp * x.ld_q * 2, s) == hipSuccess;
  void* zero5[] = {x.q, x.q_lo};
  for (void* p : zero5) ok = ok && hipMemsetAsync(p, 0, (size_t)Mp * Nq * 2, s) == hipSuccess;
  void* zero4[] = {x.hbuf, x.hbuf_lo};
  for (void* p : zero4) ok = ok && hipMemsetAsync(p, 0, (size_t)Mp * x.ld_f * 2, s) == hipSuccess;
  if (!ok) return fail(SJD_EHIP);
  // rotary table in double precision: rope[pos][i] = (cos, sin)(pos * theta^(-2i/hd))
  {
    std::vector<float2> t((size_t)x.cap_pad * (hd / 2));
    for (int p = 0; p < x.cap_pad; ++p)
      for (int i = 0; i < hd / 2; ++i) {
        const double ang = (double)p * std::pow((double)c.rope_theta, -2.0 * i / hd);
        t[(size_t)p * (hd / 2) + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
      }
    if (hipMemcpyAsync(x.rope, t.data(), t.size() * sizeof(float2), hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return fail(SJD_EHIP);
  }
  // tune the projections this process has not met yet (their consumers
  // write layer 0's cache rows 0..31 and the work planes: cleared after)
  bool tuned = false;
  for (Proj& p : projs) {
    if (!p.tune) continue;
    std::lock_guard<std::mutex> lk(g_plan_mu);
    const auto key = std::make_tuple(p.kind, p.N, p.K, p.cls);
    auto it = g_plan.find(key);
    if (it == g_plan.end()) {
      const Ctx::Plan best =
          p.cand.size() > 1 ? tune_projection(x, p.kind, p.cand, p.closed, p.cls ? 64 : 32, s) : p.cand[0];
      if (best.S < 1) return fail(SJD_EHIP);
      it = g_plan.emplace(key, best).first;
      tuned = true;
    }
    x.plan[p.cls][p.kind] = it->second;
  }
  for (int k = 0; k < 4; ++k) {
    Ctx::Plan pw = x.plan[1][k];
    const int groups = (kind_N[k] / 32 + (pw.wide ? 7 : 3)) / (pw.wide ? 8 : 4);
    const int smax_one = ncu / groups > 0 ? ncu / groups : 1;
    if (pw.S > smax_one) pw.S = smax_one;
    x.plan_wide[k] = pw;
  }
  if (tuned) {
    bool okz = hipMemsetAsync(x.x, 0, (size_t)Mp * d * sizeof(float), s) == hipSuccess;
    for (void* p : zero) okz = okz && hipMemsetAsync(p, 0, kv * 2, s) == hipSuccess;
    for (void* p : zero2) okz = okz && hipMemsetAsync(p, 0, xnsz * 2, s) == hipSuccess;
    for (void* p : zero5) okz = okz && hipMemsetAsync(p, 0, (size_t)Mp * Nq * 2, s) == hipSuccess;
    for (void* p : zero4) okz = okz && hipMemsetAsync(p, 0, (size_t)Mp * x.ld_f * 2, s) == hipSuccess;
    if (!okz || hipStreamSynchronize(s) != hipSuccess) return fail(SJD_EHIP);
  }
  if (x.use_graph && hipStreamCreateWithFlags(&x.cap_stream, hipStreamNonBlocking) != hipSuccess)
    return fail(SJD_EHIP);
  // pinned, device-visible: the step's last kernel writes the cached-row
  // counts into it directly
  if (hipHostMalloc((void**)&x.h_n, sizeof(int32_t) * kRing * x.B, hipHostMallocDefault) != hipSuccess)
    return fail(SJD_ENOMEM);
  for (int i = 0; i < kRing * x.B; ++i) x.h_n[i] = 0;
  if (hipHostGetDevicePointer((void**)&x.h_n_dev, x.h_n, 0) != hipSuccess) return fail(SJD_EHIP);
  for (int i = 0; i < kRing; ++i) {
    if (hipEventCreateWithFlags(&x.ev[i], hipEventDisableTiming) != hipSuccess) return fail(SJD_EHIP);
    x.n_events = i + 1;
    x.ev_step[i] = -1;
  }
  *out = h;
  return SJD_OK;
}

namespace {

// Caches the first n - 1 prompt tokens (windows of Mpad rows) into the caches
// of stream `cache`.
int prefill_stream(Ctx& x, const int32_t* d_prompt, int n, int cache, hipStream_t s) {
  const sjd::Streams one{sjd::kStreamsOne, 0, 0, 0, nullptr};
  const int P = Ctx::kPrefillRows;
  for (int start = 0; start < n - 1; start += P) {
    const int M = (n - 1 - start) < P ? (n - 1 - start) : P;
    HIPTRY(sjd::launch_build_prefill(d_prompt, start, M, x.win, s));
    TRY(forward(x, M, nullptr, start, nullptr, one, cache, s));
  }
  return SJD_OK;
}

// image b with prompt d_prompt into its caches (stream b; guided: stream 2b,
// and the unconditional prompt into stream 2b + 1)
int prefill(Ctx& x, int b, const int32_t* d_prompt, int n, const int32_t* d_uncond, int n_u, uint64_t seed,
            hipStream_t s) {
  x.prefilled &= ~(1u << b);
  TRY(prefill_stream(x, d_prompt, n, x.guided ? 2 * b : b, s));
  if (d_uncond) TRY(prefill_stream(x, d_uncond, n_u, 2 * b + 1, s));
  HIPTRY(sjd::launch_state_init(x.st + b, d_prompt, n, d_uncond, n_u, x.c.L, x.c.V, x.c.vis_lo, x.c.eol_id,
                                x.c.row_len, seed, s));
  x.delta[b] = d_uncond ? n_u - n : 0;
  x.prefilled |= 1u << b;
  // the image's cache-fill bound restarts; steps before this one say nothing about it
  x.img_step0[b] = x.steps;
  x.known_n[b] = n - 1;
  x.known_step[b] = x.steps - 1;
  return SJD_OK;
}

bool all_prefilled(const Ctx& x) { return x.prefilled == (1u << x.B) - 1u; }

sjd::Streams window_streams(Ctx& x) {
  if (x.nstreams > 1) return sjd::Streams{sjd::kStreamsMulti, x.c.L, x.nstreams, x.guided ? 1 : 0, x.st};
  return sjd::Streams{sjd::kStreamsOne, 0, 0, 0, nullptr};
}

// window rows: one stream of L, or stream z in rows [32 z, 32 z + L)
int window_rows(const Ctx& x) { return 32 * (x.nstreams - 1) + x.c.L; }

// A step's window build and forward into logits buffer `buf`: replayed from
// a graph captured on the first step that uses the buffer (the kernels read
// every per-step value, such as n and the window, from device state).
int step_forward(Ctx& x, int buf, float* logits, hipStream_t s) {
  const sjd::Streams sm = window_streams(x);
  auto enqueue = [&](hipStream_t q) -> int {
    HIPTRY(sjd::launch_build_window(x.st, x.win, x.c.L, x.c.K, x.c.vis_lo, sm, q));
    return forward(x, window_rows(x), &x.st->n, 0, logits, sm, 0, q);
  };
  if (!x.use_graph) return enqueue(s);
  if (!x.fwd_exec[buf]) {
    hipGraph_t g = nullptr;
    HIPTRY(hipStreamBeginCapture(x.cap_stream, hipStreamCaptureModeRelaxed));
    const int rc = enqueue(x.cap_stream);
    const hipError_t e = hipStreamEndCapture(x.cap_stream, &g);
    if (rc != SJD_OK || e != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return rc != SJD_OK ? rc : SJD_EHIP;
    }
    const hipError_t ei = hipGraphInstantiate(&x.fwd_exec[buf], g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (ei != hipSuccess) {
      x.fwd_exec[buf] = nullptr;
      return SJD_EHIP;
    }
  }
  HIPTRY(hipGraphLaunch(x.fwd_exec[buf], s));
  return SJD_OK;
}

}  // namespace

extern "C" int sjd_prefill(sjd_ctx* h, const int32_t* d_prompt, int32_t n, uint64_t seed, void* stream) {
  return sjd_prefill_image(h, 0, d_prompt, n, seed, stream);
}

extern "C" int sjd_prefill_image(sjd_ctx* h, int32_t image, const int32_t* d_prompt, int32_t n, uint64_t seed,
                                 void* stream) {
  if (!h || !d_prompt || n < 1) return SJD_EINVAL;
  Ctx& x = h->x;
  if (x.guided || image < 0 || image >= x.B) return SJD_EINVAL;
  if (n + x.c.L > x.cap) return SJD_ESTATE;
  return prefill(x, image, d_prompt, n, nullptr, 0, seed, (hipStream_t)stream);
}

extern "C" int sjd_prefill_image_cfg(sjd_ctx* h, int32_t image, const int32_t* d_prompt, int32_t n,
                                     const int32_t* d_uncond, int32_t n_u, uint64_t seed, void* stream) {
  if (!h || !d_prompt || n < 1 || !d_uncond || n_u < 1) return SJD_EINVAL;
  Ctx& x = h->x;
  if (!x.guided || image < 0 || image >= x.B) return SJD_EINVAL;
  if (n + x.c.L > x.cap || n_u + x.c.L > x.cap) return SJD_ESTATE;
  return prefill(x, image, d_prompt, n, d_uncond, n_u, seed, (hipStream_t)stream);
}

extern "C" int sjd_prefill_cfg(sjd_ctx* h, const int32_t* d_prompt, int32_t n, const int32_t* d_uncond,
                               int32_t n_u, uint64_t seed, void* stream) {
  return sjd_prefill_image_cfg(h, 0, d_prompt, n, d_uncond, n_u, seed, stream);
}

namespace sjd {
int check_verify_limits(int V, int top_k);
}

namespace {

// The caller's drafts for image `image`'s next step (sjd_set_drafts).
int set_drafts(Ctx& x, int image, const int32_t* d_draft_tok, const float* d_draft_logits, hipStream_t s) {
  const sjd_config& c = x.c;
  HIPTRY(sjd::launch_set_drafts(x.st + image, d_draft_tok, c.L, d_draft_logits != nullptr, s));
  if (d_draft_logits) {
    // the next step reads its draft rows from the buffer the step before it
    // wrote, at q_off = 0; the statistics cached with those rows no longer
    // describe them
    float* prev = x.logits[(x.steps + 1) & 1] + (size_t)image * 32 * c.V;
    HIPTRY(hipMemcpyAsync(prev, d_draft_logits, (size_t)c.L * c.V * sizeof(float), hipMemcpyDeviceToDevice, s));
    HIPTRY(hipMemsetAsync(x.stats[(x.steps + 1) & 1], 0, sizeof(sjd::RowStatsCache) * (size_t)x.B * c.L, s));
  }
  return SJD_OK;
}

// SJD_CHECK_FINITE: counts NaN / +inf among n floats at p (synchronises s);
// *bad receives whether any was found.
int check_finite(Ctx& x, const float* p, size_t n, bool* bad, hipStream_t s) {
  HIPTRY(sjd::launch_count_nonfinite(p, n, x.nonfinite, true, s));
  int32_t h = 0;
  HIPTRY(hipMemcpyAsync(&h, x.nonfinite, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  HIPTRY(hipStreamSynchronize(s));
  *bad = h != 0;
  return SJD_OK;
}

}  // namespace

extern "C" int sjd_step(sjd_ctx* h, const int32_t* d_draft_tok, const float* d_draft_logits, int32_t L, int32_t V,
                        float temperature, int32_t top_k, uint64_t seed, uint32_t step, int32_t* d_out_meta,
                        int32_t* d_out_tok, int32_t* d_out_next, void* stream) {
  if (!h || !(temperature > 0.0f) || top_k < 0) return SJD_EINVAL;
  if ((L != 0 && L != h->x.c.L) || (V != 0 && V != h->x.c.V)) return SJD_EINVAL;
  if (!d_draft_tok && d_draft_logits) return SJD_EINVAL;
  TRY(sjd::check_verify_limits(h->x.c.V, top_k));
  Ctx& x = h->x;
  if (!all_prefilled(x)) return SJD_ESTATE;
  TRY(cache_check(x));
  hipStream_t s = (hipStream_t)stream;
  const sjd_config& c = x.c;
  const bool check = (c.flags & SJD_CHECK_FINITE) != 0;
  if (d_draft_tok) {
    if (check && d_draft_logits) {
      bool bad = false;
      TRY(check_finite(x, d_draft_logits, (size_t)x.B * c.L * c.V, &bad, s));
      if (bad) return SJD_ENONFINITE;
    }
    for (int b = 0; b < x.B; ++b)
      TRY(set_drafts(x, b, d_draft_tok + (size_t)b * c.L,
                     d_draft_logits ? d_draft_logits + (size_t)b * c.L * c.V : nullptr, s));
  }
  float* cur = x.logits[x.steps & 1];
  float* prev = x.logits[(x.steps + 1) & 1];
  TRY(step_forward(x, (int)(x.steps & 1), cur, s));
  if (check) {
    bool bad = false;
    TRY(check_finite(x, cur, (size_t)logit_rows(x) * c.V, &bad, s));
    if (bad) return SJD_ENONFINITE;
  }
  // image b: logits rows from 32 b, decoder state x.st[b], Philox trial b
  const int sstate = (int)(sizeof(sjd::DevState) / sizeof(int32_t));
  const long long lstride = x.B > 1 ? 32LL * c.V : 0;
  sjd::VerifyArgs a{};
  a.B = x.B; a.L = c.L; a.V = c.V; a.K = c.K; a.D = c.D; a.top_k = top_k; a.T = temperature;
  a.flags = c.flags & (SJD_AC | SJD_PD);
  a.seed = seed; a.step = step; a.vis_lo = c.vis_lo; a.eol = c.eol_id; a.row_len = c.row_len;
  a.cur = cur; a.cur_bstride = lstride; a.draft = prev; a.draft_bstride = lstride;
  a.q_off = &x.st->q_off; a.draft_tok = x.st->spine; a.sib = x.st->sib; a.in_meta = &x.st->D_in;
  a.state_stride = sstate; a.rec = x.rec;
  if (x.use_graph) {  // (SJD_EAGER, the reference mode, recomputes every draft distribution)
    a.stats_out = x.stats[x.steps & 1];
    a.stats_in = x.stats[(x.steps + 1) & 1];
    a.stats_tag = (uint32_t)(x.steps + 2);  // zeroed entries (tag 0) never match
  }
  sjd::FinalizeOut o{};
  o.out_meta = x.st->meta; o.meta_stride = sstate; o.out_tok = x.st->tok; o.tok_stride = sstate;
  o.out_next = x.st->spine; o.next_stride = sstate; o.out_sib = x.st->sib; o.sib_stride = sstate;
  HIPTRY(sjd::launch_verify(a, o, s));
  const sjd::KvPlanes all{nullptr, nullptr, x.kc, x.kc_lo, x.vt, x.vt_lo, x.kv_elems};
  HIPTRY(sjd::launch_kv_move(x.st, all, c.n_layers, c.n_kv_heads, c.head_dim, x.cap_pad, c.K, x.nstreams, x.guided,
                             s));
  const int slot = (int)(x.steps % kRing);
  HIPTRY(sjd::launch_state_update(x.st, d_out_meta, d_out_tok, d_out_next, c.L, x.B, x.h_n_dev + slot * x.B, s));
  HIPTRY(hipEventRecord(x.ev[slot], s));
  x.ev_step[slot] = x.steps;
  x.steps += 1;
  return SJD_OK;
}

extern "C" int sjd_set_drafts(sjd_ctx* h, int32_t image, const int32_t* d_draft_tok, const float* d_draft_logits,
                              void* stream) {
  if (!h || !d_draft_tok) return SJD_EINVAL;
  Ctx& x = h->x;
  if (image < 0 || image >= x.B) return SJD_EINVAL;
  if (!(x.prefilled & (1u << image))) return SJD_ESTATE;
  return set_drafts(x, image, d_draft_tok, d_draft_logits, (hipStream_t)stream);
}

extern "C" int sjd_forward_window(sjd_ctx* h, float* d_logits, void* stream) {
  if (!h || !d_logits) return SJD_EINVAL;
  Ctx& x = h->x;
  if (!all_prefilled(x)) return SJD_ESTATE;
  TRY(cache_check(x));
  hipStream_t s = (hipStream_t)stream;
  const sjd::Streams sm = window_streams(x);
  HIPTRY(sjd::launch_build_window(x.st, x.win, x.c.L, x.c.K, x.c.vis_lo, sm, s));
  return forward(x, window_rows(x), &x.st->n, 0, d_logits, sm, 0, s);
}

extern "C" int sjd_get_plan(const sjd_ctx* h, int32_t* splits, int32_t n) {
  if (!h || !splits || n < 1) return SJD_EINVAL;
  const Ctx& x = h->x;
  int32_t v[20];
  for (int cls = 0; cls < 2; ++cls) {
    for (int k = 0; k < 4; ++k) {
      v[10 * cls + k] = x.plan[cls][k].S;
      v[10 * cls + 5 + k] = x.plan[cls][k].wide ? 8 : 4;
    }
    v[10 * cls + 4] = 1;  // LM head: unsplit, 8 column blocks per workgroup
    v[10 * cls + 9] = 8;
  }
  for (int i = 0; i < n && i < 20; ++i) splits[i] = v[i];
  return SJD_OK;
}

extern "C" void sjd_destroy(sjd_ctx* h) {
  if (!h) return;
  Ctx& x = h->x;
  (void)hipDeviceSynchronize();
  for (hipGraphExec_t& e : x.fwd_exec)
    if (e) (void)hipGraphExecDestroy(e);
  if (x.cap_stream) (void)hipStreamDestroy(x.cap_stream);
  for (void* p : x.owned) (void)hipFree(p);
  if (x.h_n) (void)hipHostFree(x.h_n);
  for (int i = 0; i < x.n_events; ++i) (void)hipEventDestroy(x.ev[i]);
  delete h;
}
