// Internal interface of the verification kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sjd {

constexpr uint32_t kFlagAC = 1u;
constexpr uint32_t kFlagPD = 2u;
constexpr uint32_t kFlagPDInline = 1u << 30;  // (internal) rows draw their own drafting candidates
constexpr long kPdInlineRows = 512;           // launches of at most this many rows do
constexpr uint32_t kFlagFullSelect = 1u << 29;  // (internal) every row takes the full-row selection
constexpr int kRecInts = 16;  // per-row record: tok, stage, 7 drafting candidates, fresh, pad
constexpr int kVerifyMaxV = 65536;  // logits per row held on chip
constexpr int kVerifyMaxK = 2048;   // kept (top-k) tokens per row when V > kVerifyMaxK

// Target-distribution statistics of one logits row (top-k / temperature
// softmax): its largest logit, the kept-set threshold (value, index), and
// the normaliser, tagged with the step that computed them.
struct RowStatsCache {
  float m, T, tau_v;
  int32_t tau_x, all, top_k;
  uint32_t tag;
  int32_t pad;
  double invZ;
};

struct VerifyArgs {
  int B, L, V, K, D, top_k;
  float T;
  uint32_t flags;
  uint64_t seed;
  uint32_t step;
  int vis_lo, eol, row_len;
  const float* cur;          // trial b, row j -> cur + b*cur_bstride + j*V (cur_bstride 0: L*V)
  long long cur_bstride;
  const float* draft;        // draft rows: trial b, spine row j -> draft + b*draft_bstride + (q_off[b]+j)*V
  long long draft_bstride;
  // per-trial inputs; with state_stride > 0 every one of them advances by
  // state_stride int32 per trial (fields of an array of decoder states),
  // otherwise by its packed size below
  const int32_t* q_off;      // [B] or NULL (= 0)
  const int32_t* draft_tok;  // [B][L]
  const int32_t* sib;        // [B][D][K-1] or NULL
  const int32_t* in_meta;    // [B][4]
  int state_stride;
  int32_t* rec;              // [B][L][kRecInts] scratch
  // A draft row is the previous step's target row of the same logits, so
  // its distribution was computed there: stats_out[b][j] receives every
  // target row's statistics tagged stats_tag, and a draft row (b, q_off + j)
  // whose stats_in entry carries stats_tag - 1 with the same temperature and
  // top_k skips its own selection (both NULL: always computed)
  RowStatsCache* stats_out;  // [B][L] or NULL
  const RowStatsCache* stats_in;
  uint32_t stats_tag;
  int32_t* out_rows;         // [B][L][2] or NULL
  float* dbg_p;              // [B][L][V] or NULL
};

struct FinalizeOut {
  int32_t* out_meta; int meta_stride;
  int32_t* out_tok;  int tok_stride;
  int32_t* out_next; int next_stride;
  int32_t* out_sib;  int sib_stride;
};

hipError_t launch_verify(const VerifyArgs& a, const FinalizeOut& o, hipStream_t s);

// Device address, on the current device, of the static record scratch of
// sjd_verify_noalloc (SJD_VERIFY_NOALLOC_MAX_ROWS rows of kRecInts words);
// looked up once per device.
hipError_t noalloc_scratch(int32_t** out);

}  // namespace sjd
