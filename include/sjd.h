/*
 * sjd.h — C ABI of the MI355X (gfx950) speculative-Jacobi step library
 * (libsjd.so), implementing the per-iteration step of SJD-PAC:
 * "SJD-PAC: Accelerating Speculative Jacobi Decoding via Proactive Drafting
 * and Adaptive Continuation" (arXiv 2603.18599).
 *
 * One step (Alg. 1 of the paper) takes the window of draft tokens X^{t-1}
 * with their draft distributions P^{t-1}, runs one parallel forward of the
 * decoder over the cached keys/values plus the window to get P^t, verifies
 * every window position by rejection sampling (Sec. 3.2), keeps verifying
 * after the first rejection (adaptive continuation, Sec. 4.2), and after a
 * rejection drafts K - 1 extra candidates at the next D positions (proactive
 * drafting, Sec. 4.1). It returns the committed tokens and the next window.
 *
 * Conventions (all entry points):
 *  - Every pointer named d_* is a device pointer (HIP global memory on the
 *    current device). Host pointers are named h_* or are config structs.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream). Work is
 *    enqueued asynchronously; outputs are valid after the stream syncs.
 *  - Arguments are checked on the host before anything is enqueued; a bad
 *    argument returns SJD_EINVAL and enqueues nothing.
 *  - Errors reported by the HIP runtime are returned as SJD_EHIP; an
 *    asynchronous kernel failure surfaces on a later call or sync.
 *  - Tokens are absolute vocabulary ids. The sampling support is the
 *    contiguous range [vis_lo, vis_lo + V); logits rows hold V fp32 values,
 *    entry x belonging to token vis_lo + x.
 *  - No entry point is thread-safe on the same context; different contexts
 *    may be used from different threads on different streams.
 *
 * Random numbers: Philox4x32-10 (Salmon et al., SC'11). Element x of stream
 * (tag, stage, row) for trial b at step s is word (x & 3) of the block at
 * counter (x >> 2, b, tag << 24 | stage << 16 | row, s) under the key
 * (seed low 32 bits, seed high 32 bits). u = (word >> 8) * 2^-24; a race key
 * is -logf(1 - u) / w. Tags: 1 accept uniforms, 2 row samples, 3 fresh tail
 * (vanilla SJD), 4 bonus token, 5 drafting candidates, 6 placeholders.
 * Sampled results therefore depend only on (seed, trial, step, row) and the
 * logits, never on launch shape.
 */
#ifndef SJD_H
#define SJD_H
#include <stdint.h>

#if defined(__GNUC__)
#define SJD_API __attribute__((visibility("default")))
#else
#define SJD_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SJD_OK = 0,
  SJD_EINVAL = -1,  /* bad argument; nothing was enqueued                       */
  SJD_ENOMEM = -2,  /* device allocation failed                                 */
  SJD_EHIP = -3,    /* HIP runtime error                                        */
  SJD_ESTATE = -4,  /* call not valid in the context's state (e.g. cache full)  */
  SJD_ENOTSUP = -5, /* valid request this build does not support                */
  SJD_ENONFINITE = -6 /* SJD_CHECK_FINITE only: a logit is NaN or +inf; the
                         verification was not enqueued                          */
} sjd_status;

/* flags */
#define SJD_AC 1u /* adaptive continuation: no break after the first rejection (Sec. 4.2) */
#define SJD_PD 2u /* proactive drafting after a rejection (Sec. 4.1)                      */
/* decoder contexts only, the reference mode: enqueue every kernel of a step
 * directly instead of replaying the step's window forward from a captured
 * HIP graph, and compute every draft row's distribution instead of reusing
 * the statistics the previous step computed for that row (the results are
 * bitwise identical; for debugging and profiling) */
#define SJD_EAGER 4u
/* decoder contexts only: the GEMM plan (how many workgroups share each
 * projection's K range) sets the summation order and therefore the rounding
 * of the logits. By default it is fixed: the plan recorded for the shape
 * (the timed choice on MI355X for the shapes this library ships plans for),
 * else a closed form, so that a seed gives the same tokens in every process.
 * SJD_TUNE times candidate plans at sjd_init instead (the first context of a
 * process that meets a projection shape times GEMM + consumer pairs; every
 * later context of the process reuses its choice): possibly faster on other
 * shapes, but the choice depends on timing, so two processes may round
 * differently. SJD_NO_TUNE forces the closed form. */
#define SJD_NO_TUNE 8u
#define SJD_TUNE 16u
/* debug: check every logits row a verification reads for NaN and +inf first
 * (-inf marks an excluded token and is allowed). The call then synchronises
 * its stream and returns SJD_ENONFINITE, with nothing verified and no state
 * changed, if one is found. sjd_verify: in sjd_verify_params.flags;
 * decoder contexts: in sjd_config.flags. */
#define SJD_CHECK_FINITE 32u
/* sjd_verify only, the reference mode of the top-k selection: every row
 * selects its kept set by histograms over the whole row instead of by the
 * candidates at or above a threshold estimated from a sample of the row. The
 * kept sets and thresholds are the same; the normalisers are summed in a
 * different order (fp64), so a decision within a few fp64 ulps of a tie can
 * differ. For tests and profiling. */
#define SJD_FULL_SELECT 64u

/* Rows (B * L) sjd_verify_noalloc can take: its record scratch is a static
 * device array of this many 64-byte records (8 MiB per device). */
#define SJD_VERIFY_NOALLOC_MAX_ROWS 131072

/* Returns a static string naming a status code. */
SJD_API const char* sjd_status_str(int status);

/* ------------------------------------------------------------------------ */
/* Standalone verification of one window per trial on given logits.
 *
 * Paper: Alg. 1 (the verification loop and drafting after it), Sec. 3.2
 * (accept a draft with probability min(1, p/q), else draw from
 * norm(max(0, p - q))), Sec. 4.1-4.2, and Theorem 2 (Appendix A.3) for rows
 * holding several candidates.
 *
 * Window layout of one trial with tree depth D_in (0 <= D_in <= D,
 * K * D_in <= L): n_s = L - (K-1) * D_in spine rows, then (K-1) * D_in
 * sibling rows. Spine row j verifies spine draft s_j; at rows j < D_in the
 * candidates are s_j and its K-1 siblings, verified in order. Sibling row
 * n_s + j*(K-1) + (k-2) is the target row after candidate k of depth j; a
 * token drawn from it is committed when that candidate is accepted.
 * Spine rows j >= n_q have no draft distribution (appended placeholders):
 * their token is drawn from p and they count as rejected.
 * The committed prefix ends at the first spine row whose own draft was not
 * accepted (first_rej); rows after it are verified anyway and carried into
 * the next window as drafts (adaptive continuation).
 *
 * p and q of a row: keep the top_k largest logits (ties: lower index first;
 * top_k = 0 or >= V keeps all), softmax of (l - max) / temperature.
 *
 * Row end tokens: when row_len > 0, the generated-token index g of row j is
 * g0 + j, and rows with g mod (row_len + 1) == row_len take eol_id, count as
 * accepted, and get no drafting candidates.
 */
typedef struct {
  int32_t B;          /* trials (independent windows), >= 1                      */
  int32_t L;          /* rows per window, 1..64                                   */
  int32_t V;          /* logits per row, 4..65536, multiple of 4                   */
  int32_t K;          /* candidates per tree depth, 1..8                          */
  int32_t D;          /* maximum tree depth, >= 0, K * D <= L                     */
  int32_t top_k;      /* >= 0; the kept set (top_k, or V when top_k is 0 or >= V)
                         may hold at most 2048 tokens (SJD_ENOTSUP otherwise)    */
  float temperature;  /* > 0                                                      */
  uint32_t flags;     /* SJD_AC | SJD_PD, optionally | SJD_CHECK_FINITE,
                         SJD_FULL_SELECT                                           */
  uint64_t seed;
  uint32_t step;      /* counter word 3 of every random stream                   */
  int32_t vis_lo;     /* token id of logits entry 0                               */
  int32_t eol_id;     /* row end token                                            */
  int32_t row_len;    /* <= 0 disables row ends                                   */
} sjd_verify_params;

typedef struct {
  const float* d_cur;        /* [B][L][V] current logits, spine rows then sibling rows   */
  const float* d_draft;      /* [B][L][V] draft logits; spine row j < n_q reads row j     */
  const int32_t* d_draft_tok;/* [B][L] spine drafts s_0 .. s_{n_s-1}                     */
  const int32_t* d_sib;      /* [B][D][K-1] siblings (-1 = none), or NULL                 */
  const int32_t* d_in_meta;  /* [B][4] { D_in, n_q, g0, 0 }                               */
  int32_t* d_out_meta;       /* [B][8] { n_c, first_rej or -1, D', n_s', n_q', accepted
                                         sibling k or 0, g0 + n_c, 0 }                   */
  int32_t* d_out_tok;        /* [B][L] committed tokens (n_c valid, rest -1)              */
  int32_t* d_out_next;       /* [B][L] next spine drafts (n_s' valid, rest -1); the next
                                step's draft row for index i < n_q' is this step's row
                                n_c + i                                                   */
  int32_t* d_out_sib;        /* [B][D][K-1] next siblings (-1 = none); may be NULL when
                                D * (K-1) == 0                                            */
  int32_t* d_out_rows;       /* [B][L][2] (token, stage) per row, or NULL: stage k >= 1
                                candidate k accepted, 0 drawn, -1 row end                 */
  float* d_dbg_p;            /* [B][L][V] probabilities p of every row, or NULL           */
} sjd_verify_io;

/* Ownership: all buffers belong to the caller and must not overlap. The
 * library keeps a grow-only scratch buffer for per-row records (B * L * 64
 * bytes) per device and stream, allocated on first use: calls on different
 * streams never share it, and growing it waits for the work its stream has
 * queued. Errors: SJD_EINVAL for
 * out-of-range parameters, NULL required pointers or misaligned logits
 * (16-byte alignment), SJD_ENOMEM, SJD_EHIP. Drafts outside the support end
 * that row's candidate list (an invalid spine draft makes the row a plain
 * draw from p); a repeated sibling ends the list too. A trial whose in_meta
 * is invalid (D_in outside [0, D], K * D_in > L, n_q outside [0, n_s]) is
 * not verified: its out_meta becomes {-1, -1, 0, ...} and its other outputs
 * are left untouched (the meta lives in device memory, so this cannot be
 * reported as a status). */
SJD_API int sjd_verify(const sjd_verify_params* params, const sjd_verify_io* io, void* stream);

/* sjd_verify for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, kernels and results, but no allocation of any kind. The
 * per-row records live in a static device array of
 * SJD_VERIFY_NOALLOC_MAX_ROWS records, one per device for the life of the
 * process; B * L above that limit returns SJD_EINVAL with nothing enqueued.
 * Every call on a device shares that device's array, so calls that overlap
 * on one device (other streams, other threads) race and must be ordered by
 * the caller; a call leaves its records behind, and none of the next call's
 * results depend on them. */
SJD_API int sjd_verify_noalloc(const sjd_verify_params* params, const sjd_verify_io* io, void* stream);

/* ------------------------------------------------------------------------ */
/* Decoder context: weights, KV cache and window state of one generation.
 *
 * The decoder is a pre-norm LLaMA-style stack (RMSNorm, rotary embeddings in
 * the rotate-half layout, grouped-query attention, SwiGLU, untied head);
 * the paper names its models (Sec. 5.1) but not their layers.
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab_size;
  int32_t vis_lo, V;     /* sampled range of the head: rows [vis_lo, vis_lo + V)       */
  int32_t max_seq;       /* KV capacity in tokens (prompt + generated + L)             */
  int32_t L, K, D;       /* window slots (1..64), candidates per depth (1..8), depth   */
  uint32_t flags;        /* SJD_AC | SJD_PD (0 = vanilla SJD; Sec. 5.3's ablation),
                            optionally | SJD_EAGER | SJD_NO_TUNE | SJD_TUNE |
                            SJD_CHECK_FINITE                                              */
  float rms_eps, rope_theta;
  int32_t eol_id, row_len;
  int32_t weights_f32;   /* 1: weights are fp32, 0: bf16                                */
  float cfg_w;           /* classifier-free guidance weight w (Sec. 5.1 uses 3); 0 = off.
                            On: every image keeps a second (unconditional) stream,
                            prefilled by sjd_prefill_cfg / sjd_prefill_image_cfg, and
                            every step samples from l_u + w (l_c - l_u); needs L <= 32
                            (SJD_ENOTSUP otherwise) */
  int32_t batch;         /* images generated together, 1 (0 reads as 1) to 4, or to 2
                            with guidance (four streams at most; SJD_ENOTSUP beyond).
                            With more than one, every step runs all images' windows in
                            one forward (one pass over the weights; stream z in rows
                            [32 z, 32 z + L)), each image with its own cache, state and
                            prompt (sjd_prefill_image), drawing from Philox trial b;
                            needs L <= 32. The paper decodes one image at a time;
                            batching serves several requests per weight pass. */
} sjd_config;

/* Device pointers, row-major [out][in] (a Linear layer's layout), bf16 or
 * fp32 as configured. sjd_init copies them into library memory (matrices
 * repacked into the GEMM tile layout, fp32 rounded to bf16), so the caller
 * may release them once sjd_init returns.
 * h_layer is a HOST array of 9 * n_layers device pointers, per layer:
 * attn_norm[d], wq[H*hd][d], wk[Hkv*hd][d], wv[Hkv*hd][d], wo[d][H*hd],
 * ffn_norm[d], wg[F][d], wu[F][d], wd[d][F]. */
typedef struct {
  const void* d_embed;        /* [vocab][d]  */
  const void* const* h_layer; /* 9 * n_layers */
  const void* d_final_norm;   /* [d]         */
  const void* d_lm_head;      /* [vocab][d]  */
} sjd_weights;

typedef struct sjd_ctx sjd_ctx;

/* Allocates the weight copies, the KV cache and the work buffers on the
 * current device; synchronises `stream` before returning. SJD_ENOTSUP for
 * head_dim other than 64 or 128, or V > 65536. */
SJD_API int sjd_init(const sjd_config* cfg, const sjd_weights* w, void* stream, sjd_ctx** out);

/* Starts a generation (Sec. 3.3: the positions of the first window are
 * initialised and appended before the first parallel forward): writes the
 * keys/values of d_prompt[0 .. n-2], makes d_prompt[n-1] the pending token
 * and fills the window with placeholders, uniform over the sampled range
 * (stream tag 6, step word 0xFFFFFFFF) and carrying no draft distribution.
 * n >= 1, n + L <= max_seq. Prompt ids should lie in [0, vocab_size); an id
 * outside it is fed to the model as token vis_lo (nothing is read outside
 * the embedding table). sjd_prefill is sjd_prefill_image for image 0. */
SJD_API int sjd_prefill(sjd_ctx* ctx, const int32_t* d_prompt, int32_t n, uint64_t seed, void* stream);

/* sjd_prefill for image `image` (0 .. batch-1) of a batched context; the
 * other image's generation is left as it is (an image can be restarted while
 * the other one continues). Every image must have been prefilled before
 * sjd_step (SJD_ESTATE otherwise). SJD_EINVAL on a guided context. */
SJD_API int sjd_prefill_image(sjd_ctx* ctx, int32_t image, const int32_t* d_prompt, int32_t n, uint64_t seed,
                              void* stream);

/* sjd_prefill for a guided context (cfg_w != 0; SJD_EINVAL otherwise, and
 * sjd_prefill is SJD_EINVAL on a guided context): d_prompt[0..n) is the
 * text prompt, d_uncond[0..n_u) the unconditional prompt, prefilled into the
 * image's unconditional stream's cache. Both streams then receive the same
 * window tokens (the unconditional stream's first pending token is
 * d_uncond[n_u-1]) at their own positions. n, n_u >= 1; n + L <= max_seq and
 * n_u + L <= max_seq. sjd_prefill_cfg is sjd_prefill_image_cfg for image 0. */
SJD_API int sjd_prefill_cfg(sjd_ctx* ctx, const int32_t* d_prompt, int32_t n, const int32_t* d_uncond,
                            int32_t n_u, uint64_t seed, void* stream);

/* sjd_prefill_cfg for image `image` (0 .. batch-1) of a guided batched
 * context (Sec. 5.1's guided sampling, several images per weight pass); the
 * other images' generations are left as they are. */
SJD_API int sjd_prefill_image_cfg(sjd_ctx* ctx, int32_t image, const int32_t* d_prompt, int32_t n,
                                  const int32_t* d_uncond, int32_t n_u, uint64_t seed, void* stream);

/* One SJD-PAC iteration (Alg. 1): takes the drafts X^{t-1} and their draft
 * distributions P^{t-1}, runs the window forward, verification, drafting and
 * KV commit, and returns the committed tokens and the next drafts X^t (whose
 * distributions P^t the context keeps for the next step).
 *  d_draft_tok: NULL = the context's own drafts (what the previous step or
 *    the prefill left); otherwise [batch][L] vocabulary ids, row j's draft
 *    (the window feeds the pending token and drafts 0 .. L-2; draft L-1 is
 *    verified, not fed), as a plain chain without drafting siblings: the
 *    same as sjd_set_drafts for every image followed by this step.
 *  d_draft_logits: with caller drafts, NULL or [batch][L][V] logits over
 *    [vis_lo, vis_lo + V), row j's draft distribution through this step's
 *    temperature / top-k softmax; NULL gives the rows no draft distribution
 *    (each row draws from its own target row, lossless whatever the drafts'
 *    origin; the context's previous rows describe its own drafts, not the
 *    caller's). Must be NULL when d_draft_tok is NULL.
 *  L, V: the context's window slots and sampled range (0 = the context's;
 *    any other value is SJD_EINVAL).
 * Outputs (device, may be NULL): d_out_meta[8] as in sjd_verify plus word
 * 7 = cached rows after the step; d_out_tok[L] committed tokens;
 * d_out_next[L] next spine drafts (-1 past n_s'); a batched context writes
 * one such block per image ([batch][8], [batch][L], [batch][L]).
 * SJD_ESTATE if a cache cannot take another window (checked against a
 * host-side upper bound). With SJD_CHECK_FINITE the call synchronises after
 * the forward and returns SJD_ENONFINITE (state unchanged) if a logit of
 * the window or of the draft rows is NaN or +inf. */
SJD_API int sjd_step(sjd_ctx* ctx, const int32_t* d_draft_tok, const float* d_draft_logits, int32_t L, int32_t V,
                     float temperature, int32_t top_k, uint64_t seed, uint32_t step, int32_t* d_out_meta,
                     int32_t* d_out_tok, int32_t* d_out_next, void* stream);

/* Replaces the drafts of image `image`'s next step with the caller's (the
 * problem statement's step takes the previous iteration's drafts X^{t-1}
 * and their distributions P^{t-1} as inputs; Alg. 1): d_draft_tok[L] are
 * vocabulary ids, row j's draft (the next window holds the pending token
 * and d_draft_tok[0 .. L-2]; row L-1's draft is verified but not fed), and
 * d_draft_logits[L][V] (may be NULL) row j's draft distribution as logits
 * over [vis_lo, vis_lo + V), taken through the step's temperature / top-k
 * softmax like the context's own. The next window is a plain chain (no
 * drafting siblings); with NULL logits no row has a draft distribution and
 * every row draws from its own (like appended placeholders). The following
 * sjd_step then verifies these drafts; its outputs, adaptive continuation,
 * drafting and KV commit are as usual, and the steps after it use the
 * context's own drafts again. Device pointers, read on `stream` (copied,
 * so the caller may reuse them once the stream passes this call). A draft
 * outside [vis_lo, vis_lo + V) is verified as no draft (its row draws from
 * p and counts as rejected); one outside [0, vocab_size) (e.g. the -1 that
 * pads d_out_next) is fed to the model as token vis_lo.
 * SJD_ESTATE before the image is prefilled. */
SJD_API int sjd_set_drafts(sjd_ctx* ctx, int32_t image, const int32_t* d_draft_tok, const float* d_draft_logits,
                           void* stream);

/* Window forward only (no verification): logits of the current window into
 * d_logits[L][V] (a guided context: the guided logits; a batched context:
 * d_logits[32 (batch - 1) + L][V], image b's rows from row 32 b). For parity
 * tests. */
SJD_API int sjd_forward_window(sjd_ctx* ctx, float* d_logits, void* stream);

/* The context's GEMM plan, written to splits[0 .. min(n, 20)): for windows
 * of up to 32 rows, [0..5) how many workgroups share the K range of the
 * QKV, O, gate|up, down and LM-head projections and [5..10) how many 32-column
 * blocks each workgroup takes (4 or 8); [10..20) the same for windows of
 * more rows (several streams, L > 32, prefill). Chosen at sjd_init (see
 * SJD_TUNE): the plan recorded for the shape, else the closed form; with
 * SJD_TUNE the process-wide timed plan; and, when the environment variable
 * SJD_SPLITS="qkv,o,gu,down" is set (each entry S or S:blocks), that plan for
 * windows of up to 32 rows (a malformed value fails sjd_init with
 * SJD_EINVAL). The environment variable SJD_QPARTS=p likewise sets how many
 * attention workgroups share one key / value head's query heads (default:
 * one per query head; p must divide n_heads / n_kv_heads, else sjd_init
 * fails with SJD_EINVAL); it leaves every result bitwise unchanged (each
 * query head's arithmetic is the same in any workgroup), whereas a plan
 * changes the logits' rounding. */
SJD_API int sjd_get_plan(const sjd_ctx* ctx, int32_t* splits, int32_t n);

SJD_API void sjd_destroy(sjd_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif
