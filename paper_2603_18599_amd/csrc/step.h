// Internal interface of the step bookkeeping kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "forward.h"

namespace sjd {
hipError_t launch_build_window(const DevState* st, Window* w, int L, int K, int vis_lo, const Streams& sm,
                               hipStream_t s);
hipError_t launch_build_prefill(const int32_t* prompt, int start, int M, Window* w, hipStream_t s);
// next window from caller drafts: chain of tok[0..L) (row j's draft), row j's
// draft distribution from row j of the draft logits when has_q
// adds the count of NaN / +inf entries of p[0 .. n) to *cnt (zeroed first when reset)
hipError_t launch_count_nonfinite(const float* p, size_t n, int32_t* cnt, bool reset, hipStream_t s);
hipError_t launch_set_drafts(DevState* st, const int32_t* tok, int L, bool has_q, hipStream_t s);
// uncond: the unconditional prompt of a guided context (its last token is
// that stream's first pending token), or NULL
hipError_t launch_state_init(DevState* st, const int32_t* prompt, int n_p, const int32_t* uncond, int n_u, int L,
                             int V, int vis_lo, int eol, int row_len, uint64_t seed, hipStream_t s);
// c.kc / c.vt hold the whole caches ([layers][Hkv][...]); q planes unused.
// ncache caches: cache z at c + z * c.sstride, driven by image z's state, or
// (guided) caches 2b, 2b + 1 by image b's, the second at positions shifted by
// its delta_u
hipError_t launch_kv_move(const DevState* st, const KvPlanes& c, int layers, int Hkv, int hd, int cap, int K,
                          int ncache, bool guided, hipStream_t s);
// B images (states st[0..B), outputs [B][8], [B][L], [B][L]); host_n[B]:
// pinned host memory that receives each image's cached rows (or NULL)
hipError_t launch_state_update(DevState* st, int32_t* out_meta, int32_t* out_tok, int32_t* out_next, int L, int B,
                               int32_t* host_n, hipStream_t s);
}  // namespace sjd
