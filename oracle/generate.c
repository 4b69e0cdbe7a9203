/* Oracle: the generation driver around the step — prefill, the window layout,
 * the KV bookkeeping after each commit ("KV cache update & backtracking",
 * Appendix B), and a tabular toy model for exact sequence-level law checks.
 *
 * Test infrastructure only (see oracle.h); shares no code with the HIP path.
 *
 * Window layout (the paper fixes a window of L verified positions per
 * forward, Sec. 3.3, and a tree of K candidates per depth for the first D
 * positions after a rejection, Sec. 4.1):
 *   slot 0            pending token c (last committed, not yet cached) at n;
 *   slot i, 1..n_s-1  spine draft s_{i-1} at position n + i;
 *   slot n_s + d(K-1) + (k-2)  sibling k of depth d at position n + 1 + d,
 *                     seeing slots 0..d and itself.
 * Row j < n_s (output of spine slot j) verifies draft s_j; the last spine
 * draft is verified but never fed. A missing sibling slot is fed token
 * vis_lo and its output is ignored.
 * After a step that commits n_c tokens, cache rows n..n+r hold the kept spine
 * slots; an accepted sibling's key/value row moves to n + r + 1; n += n_c.
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

void orc_toy_logits(const int32_t* ctx, int len, int V, uint64_t salt, float* out) {
  uint64_t h = mix64(salt ^ 0x9E3779B97F4A7C15ull);
  for (int i = 0; i < len; ++i) h = mix64(h ^ ((uint64_t)(uint32_t)ctx[i] + ((uint64_t)(i + 1) << 32)));
  h = mix64(h ^ (uint64_t)len);
  for (int v = 0; v < V; ++v) {
    uint64_t z = mix64(h + (uint64_t)(v + 1) * 0xD1B54A32D192ED03ull);
    out[v] = (float)((double)(z >> 40) * 0x1p-24) * 4.0f - 2.0f;
  }
}

static int forced_at(const orc_verify_cfg* c, long g) {
  if (c->row_len <= 0 || g < 0) return 0;
  return (g % (long)(c->row_len + 1)) == (long)c->row_len;
}

int orc_generate(const orc_gen_cfg* cfg, const int32_t* prompt, int32_t* out_tok,
                 int32_t* steps_out, int64_t* nc_hist) {
  const orc_verify_cfg* vc = &cfg->v;
  const int L = vc->L, K = vc->K, D = vc->D, V = vc->V, Km1 = vc->K - 1;
  const int np = cfg->n_prompt;
  if (np < 1 || vc->B != 1 || L < 1 || L > 64 || K < 1 || K > 8 || D < 0 || K * D > L) return -1;
  if (!cfg->mcfg && (cfg->toy_V != V || vc->vis_lo != 0)) return -1;
  const int cap = np + cfg->n_gen + 2 * L + 2;
  if (cfg->mcfg && cfg->mcfg->max_seq < cap) return -1;
  const int cfg_on = cfg->cfg_w != 0.0f;
  const int nu = cfg_on ? cfg->n_uncond : 0;
  if (cfg_on && (!cfg->mcfg || !cfg->uncond || nu < 1 || cfg->mcfg->max_seq < nu + cfg->n_gen + 2 * L + 2))
    return -1;
  int32_t* hist = (int32_t*)calloc((size_t)cap, sizeof(int32_t));
  float* cur = (float*)malloc(sizeof(float) * (size_t)L * V);
  float* prev = (float*)malloc(sizeof(float) * (size_t)L * V);
  float* dr = (float*)calloc((size_t)L * V, sizeof(float));
  int32_t* ctx = (int32_t*)malloc(sizeof(int32_t) * (size_t)(cap + L));
  int32_t spine[64], stok[64], spos[64], otok[64], onext[64], meta[4], ometa[8];
  uint64_t anc[64];
  int32_t* sib = (int32_t*)malloc(sizeof(int32_t) * (size_t)(D * Km1 + 1));
  int32_t* osib = (int32_t*)malloc(sizeof(int32_t) * (size_t)(D * Km1 + 1));
  orc_kv* kv = cfg->mcfg ? (cfg->kv ? cfg->kv : orc_kv_new(cfg->mcfg)) : NULL;
  orc_kv* kvu = cfg_on ? (cfg->kv_u ? cfg->kv_u : orc_kv_new(cfg->mcfg)) : NULL; /* unconditional stream */
  float* curu = cfg_on ? (float*)malloc(sizeof(float) * (size_t)L * V) : NULL;
  int32_t upos[64];
  int ret = -1;
  if (!hist || !cur || !prev || !dr || !ctx || !sib || !osib || (cfg->mcfg && !kv) || (cfg_on && (!kvu || !curu)))
    goto done;

  memcpy(hist, prompt, sizeof(int32_t) * (size_t)np);
  int n = np - 1; /* cached rows; hist[n] is the pending token */
  if (kv) {
    for (int s0 = 0; s0 < n; s0 += 64) {
      int M = n - s0 < 64 ? n - s0 : 64;
      for (int a = 0; a < M; ++a) {
        stok[a] = prompt[s0 + a];
        spos[a] = s0 + a;
        anc[a] = (a == 63) ? ~0ull : ((1ull << (a + 1)) - 1ull);
      }
      if (orc_forward(cfg->mcfg, cfg->w, kv, s0, stok, spos, anc, M, NULL) != 0) goto done;
    }
  }
  /* unconditional stream: its own prompt, its own rows; nu_c = its cached
   * rows, pend_u its pending token until the first step commits */
  int nu_c = nu - 1;
  int32_t pend_u = cfg_on ? cfg->uncond[nu - 1] : 0;
  if (cfg_on) {
    for (int s0 = 0; s0 < nu_c; s0 += 64) {
      int M = nu_c - s0 < 64 ? nu_c - s0 : 64;
      for (int a = 0; a < M; ++a) {
        stok[a] = cfg->uncond[s0 + a];
        spos[a] = s0 + a;
        anc[a] = (a == 63) ? ~0ull : ((1ull << (a + 1)) - 1ull);
      }
      if (orc_forward(cfg->mcfg, cfg->w, kvu, s0, stok, spos, anc, M, NULL) != 0) goto done;
    }
  }
  /* initial window: all placeholders without a draft distribution */
  int D_in = 0, n_s = L, n_q = 0;
  long g0 = 0;
  for (int i = 0; i < L; ++i) {
    if (forced_at(vc, g0 + i)) spine[i] = vc->eol_id;
    else spine[i] = vc->vis_lo + (int)(((uint64_t)orc_bits(vc->seed, ORC_TAG_INIT, 0, (uint32_t)i, 0,
                                                             0xFFFFFFFFu, 0) * (uint64_t)V) >> 32);
  }
  for (int i = 0; i < D * Km1; ++i) sib[i] = -1;
  int q_off = 0, gen = 0, step = 0;
  while (gen < cfg->n_gen && step < cfg->max_steps) {
    /* window slots */
    for (int i = 0; i < n_s; ++i) {
      stok[i] = i == 0 ? hist[n] : spine[i - 1];
      spos[i] = n + i;
      anc[i] = (i == 63) ? ~0ull : ((1ull << (i + 1)) - 1ull);
    }
    for (int d = 0; d < D_in; ++d) {
      for (int k = 2; k <= K; ++k) {
        int t = n_s + d * Km1 + (k - 2);
        int y = sib[d * Km1 + (k - 2)];
        stok[t] = y >= 0 ? y : vc->vis_lo;
        spos[t] = n + 1 + d;
        anc[t] = ((1ull << (d + 1)) - 1ull) | (1ull << t);
      }
    }
    if (kv) {
      if (orc_forward(cfg->mcfg, cfg->w, kv, n, stok, spos, anc, L, cur) != 0) goto done;
      if (cfg_on) {
        /* same window, unconditional context and positions */
        const int32_t t0 = stok[0];
        stok[0] = pend_u;
        for (int a = 0; a < L; ++a) upos[a] = spos[a] - n + nu_c;
        if (orc_forward(cfg->mcfg, cfg->w, kvu, nu_c, stok, upos, anc, L, curu) != 0) goto done;
        stok[0] = t0;
        orc_cfg_combine(cur, curu, cfg->cfg_w, (long)L * V, cur);
      }
    } else {
      for (int a = 0; a < L; ++a) {
        int len = 0;
        for (int t = 0; t < n; ++t) ctx[len++] = hist[t];
        for (int b = 0; b < L; ++b)
          if ((anc[a] >> b) & 1u) ctx[len++] = stok[b];
        orc_toy_logits(ctx, len, V, cfg->toy_salt, cur + (size_t)a * V);
      }
    }
    for (int j = 0; j < n_q; ++j)
      memcpy(dr + (size_t)j * V, prev + (size_t)(q_off + j) * V, sizeof(float) * (size_t)V);
    meta[0] = D_in; meta[1] = n_q; meta[2] = (int32_t)g0; meta[3] = 0;
    orc_verify_cfg c1 = *vc;
    c1.step = (uint32_t)step;
    orc_verify_io io;
    memset(&io, 0, sizeof(io));
    io.cur = cur; io.draft = dr; io.draft_tok = spine; io.sib = sib; io.in_meta = meta;
    io.out_meta = ometa; io.out_tok = otok; io.out_next = onext; io.out_sib = osib;
    if (orc_verify(&c1, &io) != 0) goto done;
    if (cfg->step_meta) memcpy(cfg->step_meta + (size_t)step * 8, ometa, sizeof(ometa));
    const int n_c = ometa[0], r = ometa[1], acc_k = ometa[5];
    if (kv && acc_k >= 2) orc_kv_move(kv, n + n_s + r * Km1 + (acc_k - 2), n + r + 1);
    if (cfg_on && acc_k >= 2) orc_kv_move(kvu, nu_c + n_s + r * Km1 + (acc_k - 2), nu_c + r + 1);
    for (int i = 0; i < n_c; ++i) hist[n + 1 + i] = otok[i];
    n += n_c;
    if (cfg_on && n_c > 0) {
      nu_c += n_c;
      pend_u = otok[n_c - 1];
    }
    gen += n_c;
    if (nc_hist) nc_hist[n_c] += 1;
    memcpy(spine, onext, sizeof(int32_t) * (size_t)L);
    memcpy(sib, osib, sizeof(int32_t) * (size_t)(D * Km1));
    D_in = ometa[2]; n_s = ometa[3]; n_q = ometa[4]; g0 = ometa[6];
    float* t = prev; prev = cur; cur = t;
    q_off = n_c;
    ++step;
  }
  if (out_tok) memcpy(out_tok, hist + np, sizeof(int32_t) * (size_t)gen);
  if (steps_out) *steps_out = step;
  ret = gen;
done:
  free(hist); free(cur); free(prev); free(dr); free(ctx); free(sib); free(osib); free(curu);
  if (kv != cfg->kv) orc_kv_free(kv);
  if (kvu != cfg->kv_u) orc_kv_free(kvu);
  return ret;
}

/* Many independent toy-model generations (run r uses seed seed0 + r);
 * out receives the first n_gen tokens of each run. */
int orc_generate_many(const orc_gen_cfg* cfg, const int32_t* prompt, int runs, uint64_t seed0,
                      int32_t* out, int32_t* steps, int64_t* nc_hist) {
  if (cfg->mcfg) return -1;
  const int L = cfg->v.L;
  int err = 0;
#pragma omp parallel
  {
    int64_t* h = (int64_t*)calloc((size_t)L + 2, sizeof(int64_t));
    int32_t* buf = (int32_t*)malloc(sizeof(int32_t) * (size_t)(cfg->n_gen + 2 * L + 2));
#pragma omp for schedule(static) reduction(min : err)
    for (int r = 0; r < runs; ++r) {
      orc_gen_cfg c = *cfg;
      c.v.seed = seed0 + (uint64_t)r;
      int32_t st = 0;
      int g = orc_generate(&c, prompt, buf, &st, h);
      if (g < cfg->n_gen) { err = -1; continue; }
      memcpy(out + (size_t)r * cfg->n_gen, buf, sizeof(int32_t) * (size_t)cfg->n_gen);
      if (steps) steps[r] = st;
    }
#pragma omp critical
    {
      if (nc_hist)
        for (int i = 0; i < L + 2; ++i) nc_hist[i] += h[i];
    }
    free(h);
    free(buf);
  }
  return err;
}
