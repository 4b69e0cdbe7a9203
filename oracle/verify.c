/* Oracle: one SJD-PAC verification step (Alg. 1 of the paper) over a batch of
 * independent trials.
 *
 * Test infrastructure only (see oracle.h); shares no code with the HIP path.
 *
 * What each piece follows:
 *  - top-k / temperature softmax: the sampler settings of the experiments
 *    (top-2000 logits, temperature 1; Sec. 5.1);
 *  - accept/reject and residual: rejection sampling as stated in Sec. 3.2 and
 *    the Rejection Sampling Lemma (Appendix A.1): accept draft x with
 *    probability min(1, p(x)/q(x)), else draw from norm(max(0, p - q));
 *  - adaptive continuation: Sec. 4.2 and the "no break" loop of Alg. 1 —
 *    every spine row is verified with its own (stale) p and q, the first
 *    rejected row index is remembered, and rows after it are kept only as
 *    drafts for the next step;
 *  - several candidates at a row: Theorem 2 (Appendix A.3), candidates
 *    verified in order against p^(k) and q^(k), where q^(k) is q with the
 *    earlier candidates removed and renormalised and
 *    p^(k+1) = norm(max(0, p^(k) - q^(k))); after all are rejected a token is
 *    drawn from the last residual;
 *  - proactive drafting: Sec. 4.1 — after a rejection, the next window gets
 *    K - 1 extra candidates drawn without replacement from the current target
 *    rows at the first D positions past the commit point, next to the
 *    continued spine (first-path-pruned tree: spine plus K - 1 siblings per
 *    depth, so the number of window slots stays L);
 *  - vanilla SJD (AC off): Sec. 3.3 — the tail after the first rejection is
 *    redrawn fresh from its target rows.
 * Readings where the paper is silent (row/slot mapping, placeholders for
 * appended positions, bonus token after an accepted sibling, the race
 * sampler, forced row-end tokens) are stated next to the code that takes
 * them.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  float val;
  int idx;
} vi_t;

/* (value descending, index ascending) */
static int cmp_desc(const void* a, const void* b) {
  const vi_t* x = (const vi_t*)a;
  const vi_t* y = (const vi_t*)b;
  if (x->val > y->val) return -1;
  if (x->val < y->val) return 1;
  return (x->idx > y->idx) - (x->idx < y->idx);
}

/* Marks the top-k set of a row: the k largest logits by (value descending,
 * index ascending); k = V when top_k <= 0 or top_k >= V. */
static int topk_members(const float* logits, int V, int top_k, uint8_t* in) {
  int k = (top_k <= 0 || top_k >= V) ? V : top_k;
  vi_t* s = (vi_t*)malloc(sizeof(vi_t) * (size_t)V);
  if (!s) return -1;
  for (int x = 0; x < V; ++x) { s[x].val = logits[x]; s[x].idx = x; in[x] = 0; }
  qsort(s, (size_t)V, sizeof(vi_t), cmp_desc);
  for (int i = 0; i < k; ++i) in[s[i].idx] = 1;
  free(s);
  return 0;
}

int orc_topk_softmax(const float* logits, int V, int top_k, float T, float* p) {
  if (V < 1 || !(T > 0.0f) || top_k < 0) return -1;
  uint8_t* in = (uint8_t*)calloc((size_t)V, 1);
  if (!in || topk_members(logits, V, top_k, in) != 0) { free(in); return -1; }
  float m = -INFINITY;
  for (int x = 0; x < V; ++x)
    if (in[x] && logits[x] > m) m = logits[x];
  double Z = 0.0;
  for (int x = 0; x < V; ++x) {
    if (in[x]) {
      float d = logits[x] - m;
      float a = d / T;
      float w = expf(a);
      p[x] = w;
      Z += (double)w;
    } else {
      p[x] = 0.0f;
    }
  }
  for (int x = 0; x < V; ++x)
    if (in[x]) p[x] = (float)((double)p[x] / Z);
  free(in);
  return 0;
}

int orc_topk_rank(const float* logits, int V, int top_k, int* rank) {
  if (V < 1 || top_k < 0) return -1;
  uint8_t* in = (uint8_t*)calloc((size_t)V, 1);
  if (!in || topk_members(logits, V, top_k, in) != 0) { free(in); return -1; }
  int r = 0;
  for (int x = 0; x < V; ++x) rank[x] = in[x] ? r++ : -1;
  free(in);
  return 0;
}

/* Row end rule (not in the paper; the image-token layouts of the benchmark
 * models end each row of W image tokens with a fixed token): generated index
 * g is forced iff g mod (W + 1) == W. */
static int is_forced(const orc_verify_cfg* c, long g) {
  if (c->row_len <= 0 || g < 0) return 0;
  return (g % (long)(c->row_len + 1)) == (long)c->row_len;
}

static float fminf_(float a, float b) { return a < b ? a : b; }

typedef struct {
  int tok;      /* outcome token (local index), or -1 when forced          */
  int stage;    /* k >= 1: candidate k accepted; 0: drawn by a race; -1 forced */
  float m_acc;  /* min |u - ratio| over the accept tests taken             */
  float m_race; /* relative key gap of the race taken                      */
  float m_cond; /* residual conditioning r(x) / max(p(x), q(x)) of winner  */
} row_out;

/* Verification of one spine row with candidate list cand[0..nc) (distinct,
 * in range) against target p and draft q (Theorem 2; K = 1 is the plain
 * single-draft test of Sec. 3.2). */
static void verify_row(const orc_verify_cfg* c, const float* p, const float* q, const int* rank,
                       const int* cand, int ncand, uint32_t row, uint32_t trial,
                       float* rho, float* rho_new, uint8_t* excl, row_out* out) {
  const int V = c->V;
  out->m_acc = INFINITY;
  out->m_race = INFINITY;
  out->m_cond = INFINITY;
  memcpy(rho, p, sizeof(float) * (size_t)V);
  memset(excl, 0, (size_t)V);
  float Nf = 1.0f;   /* p^(1) = p as given, no renormalisation */
  float Qsum = 0.0f; /* q mass of the candidates already rejected */
  int tried = 0;
  for (int k = 1; k <= ncand; ++k) {
    int x = cand[k - 1];
    float den = 1.0f - Qsum;
    float pk = rho[x] / Nf;
    float qk = (den > 0.0f) ? q[x] / den : 0.0f;
    float u = orc_uniform(orc_bits(c->seed, ORC_TAG_ACC, (uint32_t)(k - 1), row, trial, c->step, 0));
    int acc;
    if (qk > 0.0f) {
      float ratio = pk / qk;
      acc = u < ratio;
      out->m_acc = fminf_(out->m_acc, fabsf(u - ratio));
    } else {
      acc = pk > 0.0f;
    }
    tried = k;
    if (acc) {
      out->tok = x;
      out->stage = k;
      return;
    }
    /* residual p^(k+1) (unnormalised) = max(0, p^(k) - q^(k)); q^(k) is zero
     * on the candidates rejected before stage k */
    double Nd = 0.0;
    for (int y = 0; y < V; ++y) {
      float py = rho[y] / Nf;
      float qy = (excl[y] || !(den > 0.0f)) ? 0.0f : q[y] / den;
      float r = py - qy;
      rho_new[y] = r > 0.0f ? r : 0.0f;
      Nd += (double)rho_new[y];
    }
    excl[x] = 1;
    Qsum = Qsum + q[x];
    if (!(Nd > 0.0)) break; /* rounding left no residual mass: draw from p^(k) */
    memcpy(rho, rho_new, sizeof(float) * (size_t)V);
    Nf = (float)Nd;
  }
  float gap;
  int t = orc_race_ranked(rho, rank, V, c->seed, ORC_TAG_RES, (uint32_t)tried, row, trial, c->step, &gap);
  out->tok = t;
  out->stage = 0;
  out->m_race = gap;
  if (t >= 0 && tried > 0) {
    float mx = p[t] > q[t] ? p[t] : q[t];
    out->m_cond = mx > 0.0f ? rho[t] / Nf / mx : INFINITY;
  }
}

/* K - 1 siblings for the next window: the K - 1 smallest race keys of p over
 * its support without token excl_tok, ascending (a draw of K - 1 tokens
 * without replacement from p restricted to the other tokens). */
static void pd_siblings(const orc_verify_cfg* c, const float* p, const int* rank, int excl_tok, uint32_t row,
                        uint32_t trial, int* sib, float* m_gap) {
  orc_race_topn_ranked(p, rank, c->V, c->K - 1, excl_tok, c->seed, ORC_TAG_PD, 0, row, trial, c->step, sib,
                       m_gap);
}

static int verify_trial(const orc_verify_cfg* c, const orc_verify_io* io, int b) {
  const int L = c->L, V = c->V, K = c->K, D = c->D;
  const int Km1 = K - 1;
  const int32_t* meta = io->in_meta + 4 * (size_t)b;
  const int D_in = meta[0], n_q = meta[1];
  const long g0 = meta[2];
  if (D_in < 0 || D_in > D || K * D_in > L) return -1;
  const int n_s = L - Km1 * D_in;
  if (n_q < 0 || n_q > n_s) return -1;
  const float* cur = io->cur + (size_t)b * L * V;
  const float* dra = io->draft + (size_t)b * L * V;
  const int32_t* s = io->draft_tok + (size_t)b * L;
  const int32_t* sib = io->sib ? io->sib + (size_t)b * D * Km1 : NULL;
  const int eol = c->eol_id;
  const uint32_t tr = c->trial0 + (uint32_t)b; /* counter word 1 */

  float* P = (float*)malloc(sizeof(float) * (size_t)L * V);
  float* Q = (float*)malloc(sizeof(float) * (size_t)V);
  float* rho = (float*)malloc(sizeof(float) * (size_t)V);
  float* rho2 = (float*)malloc(sizeof(float) * (size_t)V);
  uint8_t* excl = (uint8_t*)malloc((size_t)V);
  row_out* ro = (row_out*)calloc((size_t)L, sizeof(row_out));
  int* fresh = (int*)malloc(sizeof(int) * (size_t)L);
  int* pds = (int*)malloc(sizeof(int) * (size_t)L * (Km1 > 0 ? Km1 : 1));
  float* pdgap = (float*)malloc(sizeof(float) * (size_t)L);
  int* R = (int*)malloc(sizeof(int) * (size_t)L * V);
  if (!P || !Q || !rho || !rho2 || !excl || !ro || !fresh || !pds || !pdgap || !R) {
    free(P); free(Q); free(rho); free(rho2); free(excl); free(ro); free(fresh); free(pds); free(pdgap); free(R);
    return -2;
  }
  /* p of every row, and the rank of each kept token in its row's top-k set
   * (index order): races of a row take the stream element of that rank */
  for (int j = 0; j < L; ++j) {
    orc_topk_softmax(cur + (size_t)j * V, V, c->top_k, c->T, P + (size_t)j * V);
    orc_topk_rank(cur + (size_t)j * V, V, c->top_k, R + (size_t)j * V);
  }
  if (io->dbg_p) memcpy(io->dbg_p + (size_t)b * L * V, P, sizeof(float) * (size_t)L * V);

  /* ---- spine rows: row j is the output of the slot that feeds the token
   * before s_j, i.e. p_j = P^t(. | X_{<j}) verifies draft s_j. */
  for (int j = 0; j < n_s; ++j) {
    const float* p = P + (size_t)j * V;
    const int* rk = R + (size_t)j * V;
    row_out* o = &ro[j];
    o->m_acc = o->m_race = o->m_cond = INFINITY;
    int* my_sib = pds + (size_t)j * (Km1 > 0 ? Km1 : 1);
    for (int i = 0; i < Km1; ++i) my_sib[i] = -1;
    pdgap[j] = INFINITY;
    if (is_forced(c, g0 + j)) {
      o->tok = -1; o->stage = -1; fresh[j] = -1;
      continue;
    }
    if (j >= n_q) {
      /* appended placeholder with no draft distribution: its token is drawn
       * from p directly and the row counts as rejected (stage-0 stream). */
      float gap;
      o->tok = orc_race_ranked(p, rk, V, c->seed, ORC_TAG_RES, 0, (uint32_t)j, tr, c->step, &gap);
      o->stage = 0;
      o->m_race = gap;
    } else {
      orc_topk_softmax(dra + (size_t)j * V, V, c->top_k, c->T, Q);
      int cand[16];
      int nc = 0;
      int x0 = s[j] - c->vis_lo;
      if (x0 >= 0 && x0 < V) {
        cand[nc++] = x0;
        if (j < D_in && sib) {
          for (int k = 0; k < Km1; ++k) {
            int y = sib[(size_t)j * Km1 + k];
            if (y < 0) break;
            y -= c->vis_lo;
            int dup = (y < 0 || y >= V);
            for (int t = 0; t < nc && !dup; ++t) dup = (cand[t] == y);
            if (dup) break; /* a repeated or out-of-range candidate ends the list */
            cand[nc++] = y;
          }
        }
      }
      if (nc == 0) {
        float gap;
        o->tok = orc_race_ranked(p, rk, V, c->seed, ORC_TAG_RES, 0, (uint32_t)j, tr, c->step, &gap);
        o->stage = 0;
        o->m_race = gap;
      } else {
        verify_row(c, p, Q, rk, cand, nc, (uint32_t)j, tr, rho, rho2, excl, o);
      }
    }
    if (!(c->flags & ORC_AC)) {
      float gap;
      fresh[j] = orc_race_ranked(p, rk, V, c->seed, ORC_TAG_FRESH, 0, (uint32_t)j, tr, c->step, &gap);
      o->m_race = fminf_(o->m_race, gap);
    } else {
      fresh[j] = o->tok;
    }
    if ((c->flags & ORC_PD) && Km1 > 0) {
      int spine_next = (c->flags & ORC_AC) ? o->tok : fresh[j];
      pd_siblings(c, p, rk, spine_next, (uint32_t)j, tr, my_sib, &pdgap[j]);
    }
  }

  /* ---- sibling rows: the output after sibling (d, k) is a bonus draw used
   * only if that sibling is accepted (its own slot sees the exact prefix). */
  for (int d = 0; d < D_in; ++d) {
    for (int k = 2; k <= K; ++k) {
      int t = n_s + d * Km1 + (k - 2);
      row_out* o = &ro[t];
      o->m_acc = o->m_race = o->m_cond = INFINITY;
      int y = sib ? sib[(size_t)d * Km1 + (k - 2)] : -1;
      if (y < 0 || is_forced(c, g0 + d)) { o->tok = -1; o->stage = 0; continue; }
      if (is_forced(c, g0 + d + 1)) { o->tok = -1; o->stage = -1; continue; }
      float gap;
      o->tok = orc_race_ranked(P + (size_t)t * V, R + (size_t)t * V, V, c->seed, ORC_TAG_BONUS, 0, (uint32_t)t, tr,
                               c->step, &gap);
      o->stage = 0;
      o->m_race = gap;
    }
  }

  /* ---- finalize: first_rej_idx is the first spine row whose own draft was
   * not accepted (Alg. 1); everything before it, plus that row's outcome, is
   * committed. An accepted sibling commits itself and its bonus token. */
#define TOKOF(o) ((o).stage == -1 ? eol : (o).tok + c->vis_lo)
  int32_t* otok = io->out_tok + (size_t)b * L;
  for (int j = 0; j < L; ++j) otok[j] = -1;
  int r = -1;
  for (int j = 0; j < n_s; ++j) {
    int accepted = (ro[j].stage == -1) || (ro[j].stage == 1);
    if (!accepted) { r = j; break; }
  }
  int n_c, acc_k = 0;
  if (r < 0) {
    n_c = n_s;
    for (int j = 0; j < n_s; ++j) otok[j] = TOKOF(ro[j]);
  } else {
    for (int j = 0; j < r; ++j) otok[j] = TOKOF(ro[j]);
    if (ro[r].stage >= 2) {
      acc_k = ro[r].stage;
      int t = n_s + r * Km1 + (acc_k - 2);
      otok[r] = ro[r].tok + c->vis_lo;
      otok[r + 1] = TOKOF(ro[t]);
      n_c = r + 2;
    } else {
      otok[r] = TOKOF(ro[r]);
      n_c = r + 1;
    }
  }

  /* ---- next window: rows after the commit point become the next drafts
   * (their q row is this step's p row at the same position); positions past
   * this window are appended as placeholders without a draft distribution. */
  int Dn = 0;
  if ((c->flags & ORC_PD) && r >= 0 && Km1 > 0) {
    Dn = D;
    if (n_s - n_c < Dn) Dn = n_s - n_c;
    if (L / K < Dn) Dn = L / K;
    if (Dn < 0) Dn = 0;
  }
  const int n_s2 = L - Km1 * Dn;
  int n_q2 = n_s - n_c;
  if (n_q2 < 0) n_q2 = 0;
  if (n_q2 > n_s2) n_q2 = n_s2;
  int32_t* onext = io->out_next + (size_t)b * L;
  int32_t* osib = io->out_sib + (size_t)b * D * Km1;
  for (int i = 0; i < L; ++i) onext[i] = -1;
  for (int i = 0; i < D * Km1; ++i) osib[i] = -1;
  for (int i = 0; i < n_s2; ++i) {
    int j = n_c + i;
    long g = g0 + n_c + i;
    if (j < n_s) {
      if (ro[j].stage == -1) onext[i] = eol;
      else onext[i] = ((c->flags & ORC_AC) ? ro[j].tok : fresh[j]) + c->vis_lo;
    } else if (is_forced(c, g)) {
      onext[i] = eol;
    } else {
      uint32_t bits = orc_bits(c->seed, ORC_TAG_INIT, 0, (uint32_t)i, tr, c->step, 0);
      onext[i] = c->vis_lo + (int)(((uint64_t)bits * (uint64_t)V) >> 32);
    }
  }
  for (int d = 0; d < Dn; ++d) {
    int j = n_c + d;
    if (ro[j].stage == -1) continue;
    for (int k = 0; k < Km1; ++k) {
      int y = pds[(size_t)j * Km1 + k];
      osib[(size_t)d * Km1 + k] = y < 0 ? -1 : y + c->vis_lo;
    }
  }
  int32_t* om = io->out_meta + 8 * (size_t)b;
  om[0] = n_c; om[1] = r; om[2] = Dn; om[3] = n_s2; om[4] = n_q2; om[5] = acc_k;
  om[6] = (int32_t)(g0 + n_c); om[7] = 0;

  if (io->out_rows) {
    int32_t* orow = io->out_rows + (size_t)b * L * 2;
    for (int j = 0; j < L; ++j) {
      int used = (j < n_s) || (j - n_s) < D_in * Km1;
      orow[2 * j] = used ? (ro[j].stage == -1 ? eol : (ro[j].tok < 0 ? -1 : ro[j].tok + c->vis_lo)) : -1;
      orow[2 * j + 1] = used ? ro[j].stage : 0;
    }
  }
  if (io->out_margin) {
    float* om2 = io->out_margin + (size_t)b * L * 4;
    for (int j = 0; j < L; ++j) {
      om2[4 * j + 0] = ro[j].m_acc;
      om2[4 * j + 1] = ro[j].m_race;
      om2[4 * j + 2] = j < n_s ? pdgap[j] : INFINITY;
      om2[4 * j + 3] = ro[j].m_cond;
    }
  }
#undef TOKOF
  free(P); free(Q); free(rho); free(rho2); free(excl); free(ro); free(fresh); free(pds); free(pdgap); free(R);
  return 0;
}

int orc_verify(const orc_verify_cfg* c, const orc_verify_io* io) {
  if (!c || !io || c->B < 1 || c->L < 1 || c->L > 64 || c->V < 1 || c->K < 1 || c->K > 8 ||
      c->D < 0 || c->K * c->D > c->L || !(c->T > 0.0f) || c->top_k < 0)
    return -1;
  if (!io->cur || !io->draft || !io->draft_tok || !io->in_meta || !io->out_meta || !io->out_tok ||
      !io->out_next || !io->out_sib)
    return -1;
  int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(min : err)
  for (int b = 0; b < c->B; ++b) {
    int e = verify_trial(c, io, b);
    if (e < err) err = e;
  }
  return err;
}
