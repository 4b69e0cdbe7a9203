/*
 * Oracle for the SJD-PAC speculative Jacobi step: plain, slow, obviously
 * correct CPU code.
 *
 * THIS IS TEST INFRASTRUCTURE. Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load it. The product path (the HIP
 * library) never links, loads or calls anything in here, and nothing in here
 * includes any header of the HIP library: the two implementations share no
 * code. They share only the written rules below, restated from the paper.
 *
 * Paper: "SJD-PAC: Accelerating Speculative Jacobi Decoding via Proactive
 * Drafting and Adaptive Continuation" (arXiv 2603.18599).
 *
 * Precision. Verification decisions are taken in fp32 (the precision of the
 * GPU kernel; the paper fixes none), with fp64 used only for the softmax
 * normaliser and residual masses. The transformer forward accumulates in
 * fp64 over bf16 weights converted exactly to fp32.
 *
 * Tokens are absolute ids. The sampling support is [vis_lo, vis_lo + V);
 * logits rows hold V entries, entry x being token vis_lo + x.
 */
#ifndef SJD_ORACLE_H
#define SJD_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------- counter-based random numbers (Philox4x32-10) -------------------
 * Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
 * SC'11. Ten rounds of the 4x32 Philox bijection, key schedule bumped by the
 * Weyl constants between rounds. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Stream tags. The counter of element x of stream (tag, stage, row) for trial
 * b at step s is (x >> 2, b, tag << 24 | stage << 16 | row, s), the key is the
 * 64-bit seed split into (low, high) words, and the word used is lane x & 3. */
enum {
  ORC_TAG_ACC = 1,   /* acceptance uniforms, one per (row, stage)          */
  ORC_TAG_RES = 2,   /* races that produce a row's sampled token           */
  ORC_TAG_FRESH = 3, /* vanilla-SJD fresh tail samples                     */
  ORC_TAG_BONUS = 4, /* token after an accepted sibling                    */
  ORC_TAG_PD = 5,    /* proactive-drafting sibling candidates              */
  ORC_TAG_INIT = 6   /* placeholders for appended window positions         */
};
uint32_t orc_bits(uint64_t seed, uint32_t tag, uint32_t stage, uint32_t row,
                  uint32_t trial, uint32_t step, uint32_t x);
/* u = (bits >> 8) * 2^-24, in [0, 1). */
float orc_uniform(uint32_t bits);
/* Exp(1) variate -log(1 - u). */
float orc_exp1(uint32_t bits);

/* ---------- top-k / temperature softmax ------------------------------------
 * S = the k largest logits ordered by (value descending, index ascending);
 * k = V when top_k <= 0 or top_k >= V. w_x = expf((l_x - m) / T) on S with m
 * the largest logit, Z = sum of w in fp64, p_x = (float)(w_x / Z); p_x = 0
 * off S. Returns 0, or -1 on bad arguments. */
int orc_topk_softmax(const float* logits, int V, int top_k, float T, float* p);
/* rank[x] = position of x among the kept (top-k) tokens in index order, -1
 * for tokens outside the set. */
int orc_topk_rank(const float* logits, int V, int top_k, int* rank);

/* Exponential race: argmin over x with w_x > 0 of E_x / w_x (fp32 division),
 * E_x from stream (tag, stage, row); equal keys go to the smaller index.
 * Returns -1 when no weight is positive. If gap != NULL it receives the
 * relative gap between the best and second-best keys (1 if only one). */
int orc_race(const float* w, int V, uint64_t seed, uint32_t tag, uint32_t stage,
             uint32_t row, uint32_t trial, uint32_t step, float* gap);
/* The same race with the exponential of token x taken from element rank[x]
 * of the stream instead of element x (rank may be NULL: rank[x] = x). The
 * verification step uses rank = position of x in the row's top-k set in
 * index order, so the races of a row draw one stream element per kept
 * token. */
int orc_race_ranked(const float* w, const int* rank, int V, uint64_t seed, uint32_t tag,
                    uint32_t stage, uint32_t row, uint32_t trial, uint32_t step, float* gap);

/* The n smallest race keys (n <= 16) among tokens x != excl with w_x > 0, in
 * ascending key order, ties to the smaller index: a draw of n tokens without
 * replacement from w (the successive-sampling law). out[n] is padded with -1;
 * returns the number found. gap receives the smallest relative gap between
 * consecutive keys among the n + 1 smallest. */
int orc_race_topn(const float* w, int V, int n, int excl, uint64_t seed, uint32_t tag,
                  uint32_t stage, uint32_t row, uint32_t trial, uint32_t step, int* out,
                  float* gap);
int orc_race_topn_ranked(const float* w, const int* rank, int V, int n, int excl, uint64_t seed,
                         uint32_t tag, uint32_t stage, uint32_t row, uint32_t trial, uint32_t step,
                         int* out, float* gap);
/* trials independent races (trial b = counter word 1): out[trials] for n <= 1,
 * else the n smallest keys of each, out[trials][n]. */
void orc_race_many(const float* w, int V, int n, uint64_t seed, uint32_t tag, uint32_t stage,
                   uint32_t row, uint32_t step, int trials, int* out);
/* the same with the exponential of token x taken from element rank[x] (the
 * ranked races above; rank may be NULL) */
void orc_race_many_ranked(const float* w, const int* rank, int V, int n, uint64_t seed, uint32_t tag,
                          uint32_t stage, uint32_t row, uint32_t step, int trials, int* out);

/* ---------- one verification step over a batch of independent trials ------ */

/* flags */
#define ORC_AC 1u        /* adaptive continuation (no break)             */
#define ORC_PD 2u        /* proactive drafting                           */

typedef struct {
  int32_t B, L, V, K, D, top_k;
  float T;
  uint32_t flags;
  uint64_t seed;
  uint32_t step;
  int32_t vis_lo;    /* token id of logits entry 0                         */
  int32_t eol_id;    /* forced row-end token                               */
  int32_t row_len;   /* image tokens per row; <= 0 disables forcing        */
  uint32_t trial0;   /* counter word 1 of trial b is trial0 + b              */
} orc_verify_cfg;

/* Per-trial input meta, int32[4]: { D_in, n_q, g0, 0 }.
 *   D_in : tree depth of this window (siblings at spine rows 0..D_in-1);
 *   n_q  : spine rows 0..n_q-1 carry a draft distribution (q row), later
 *          spine rows are placeholders without one;
 *   g0   : generated-token index of the position row 0 predicts (for the
 *          forced row-end rule; ignored when row_len <= 0).
 * Per-trial output meta, int32[8]:
 *   { n_c, first_rej (-1: none), D', n_s', n_q', acc_k (0: none), g0', 0 }. */
typedef struct {
  const float* cur;         /* [B][L][V] current logits (spine then sibling rows) */
  const float* draft;       /* [B][L][V] draft logits, spine row j uses row j     */
  const int32_t* draft_tok; /* [B][L] spine drafts s_0..s_{n_s-1}                 */
  const int32_t* sib;       /* [B][D][K-1] siblings, -1 = none; NULL = none       */
  const int32_t* in_meta;   /* [B][4]                                             */
  int32_t* out_meta;        /* [B][8]                                             */
  int32_t* out_tok;         /* [B][L] committed tokens, n_c valid, rest -1        */
  int32_t* out_next;        /* [B][L] next spine drafts, n_s' valid, rest -1      */
  int32_t* out_sib;         /* [B][D][K-1] next siblings, -1 = none               */
  int32_t* out_rows;        /* [B][L][2] per row (token, stage) or NULL           */
  float* out_margin;        /* [B][L][4] per row decision margins or NULL         */
  float* dbg_p;             /* [B][L][V] p of every row or NULL                   */
} orc_verify_io;

int orc_verify(const orc_verify_cfg* cfg, const orc_verify_io* io);

/* ---------- transformer window forward ------------------------------------ */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim;
  int32_t vocab_size, vis_lo, V; /* logits cover lm_head rows [vis_lo, vis_lo+V) */
  int32_t max_seq;
  float rms_eps, rope_theta;
} orc_model_cfg;

/* bf16 weights as raw uint16 words, row-major [out][in] like a Linear layer.
 * layer[l] points at 9 arrays: attn_norm[d], wq[H*hd][d], wk[Hkv*hd][d],
 * wv[Hkv*hd][d], wo[d][H*hd], ffn_norm[d], wg[F][d], wu[F][d], wd[d][F].
 * If is_f32 is set every array holds float instead. */
typedef struct {
  const void* embed;       /* [vocab][d] */
  const void* const* layer;/* n_layers * 9 pointers */
  const void* final_norm;  /* [d] */
  const void* lm_head;     /* [vocab][d] */
  int32_t is_f32;
} orc_weights;

typedef struct orc_kv orc_kv;
orc_kv* orc_kv_new(const orc_model_cfg* cfg);
void orc_kv_free(orc_kv* kv);
/* Copy cache row src to row dst in every layer. */
void orc_kv_move(orc_kv* kv, int src, int dst);
/* Key and value row `row` of layer `layer` (Hkv*hd doubles each, rotary
 * already applied to the key), for inspection by the tests. */
void orc_kv_row(const orc_kv* kv, int layer, int row, double* k, double* v);

/* M slots; slot a holds token tok[a] at position pos[a]; it attends to cache
 * rows [0, n) and to window slot b iff bit b of anc[a] is set (anc[a] must
 * include a itself). The window's keys and values are written to cache rows
 * n .. n+M-1 in slot order. logits (M x V) may be NULL to skip the head.
 * Returns 0, -1 on bad arguments. */
int orc_forward(const orc_model_cfg* cfg, const orc_weights* w, orc_kv* kv, int n,
                const int32_t* tok, const int32_t* pos, const uint64_t* anc, int M,
                float* logits);

/* ---------- classifier-free guidance ----------------------------------------
 * The paper samples with a CFG weight of 3 (Sec. 5.1). Reading: the standard
 * logit-space guidance of autoregressive image models, l = l_u + w (l_c - l_u)
 * with l_c the logits under the text prompt and l_u under the unconditional
 * prompt, evaluated in fp64 and rounded once; the guided logits are what is
 * sampled and what the next step's drafts are verified against. */
void orc_cfg_combine(const float* l_c, const float* l_u, float w, long n, float* out);

/* ---------- generation driver (prefill + repeated steps) ------------------- */

/* Tabular toy model over V tokens: the logits of a slot are a hash of its
 * whole context (every token before it and its own token), mapped to
 * [-2, 2). Used for exact sequence-level law checks. */
void orc_toy_logits(const int32_t* ctx, int len, int V, uint64_t salt, float* out);

typedef struct {
  orc_verify_cfg v;          /* B must be 1 */
  int32_t n_prompt;
  int32_t n_gen;             /* stop after this many committed tokens */
  int32_t max_steps;
  /* model: exactly one of these */
  const orc_model_cfg* mcfg; const orc_weights* w;   /* transformer */
  int32_t toy_V; uint64_t toy_salt;                  /* toy model (mcfg NULL) */
  /* classifier-free guidance (transformer only): weight cfg_w != 0 enables
   * a second, unconditional stream with its own cache, prefilled from
   * uncond[0..n_uncond); its window holds the same tokens (its first
   * pending token is uncond[n_uncond-1]) at its own positions. */
  float cfg_w;
  const int32_t* uncond;
  int32_t n_uncond;
  /* optional, for inspection (NULL: unused): step_meta[max_steps][8]
   * receives every step's verification out-meta; kv (and kv_u, the
   * unconditional stream's) is a cache made by orc_kv_new that the driver
   * uses instead of allocating its own, so that it holds the final cache
   * when the generation returns */
  int32_t* step_meta;
  orc_kv* kv;
  orc_kv* kv_u;
} orc_gen_cfg;

/* Generates up to n_gen tokens after prompt[0..n_prompt). out_tok receives
 * the committed tokens (n_gen + L slack), steps_out the number of steps,
 * nc_hist[L+2] (may be NULL) the histogram of n_c. The seed of cfg->v is the
 * generation seed; step t uses counter word t. Returns number of generated
 * tokens, or -1 on error. */
int orc_generate(const orc_gen_cfg* cfg, const int32_t* prompt, int32_t* out_tok,
                 int32_t* steps_out, int64_t* nc_hist);

/* runs independent toy-model generations in parallel, run r with seed
 * seed0 + r; out[runs][n_gen], steps[runs] (may be NULL), nc_hist[L+2]
 * accumulated (may be NULL). Returns 0 or -1. */
int orc_generate_many(const orc_gen_cfg* cfg, const int32_t* prompt, int runs, uint64_t seed0,
                      int32_t* out, int32_t* steps, int64_t* nc_hist);

#ifdef __cplusplus
}
#endif
#endif
