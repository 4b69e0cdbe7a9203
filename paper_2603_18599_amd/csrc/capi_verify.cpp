// C ABI: status strings and the standalone verification entry point.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>
#include <utility>

#include "sjd.h"
#include "step.h"
#include "verify.h"

namespace {

// Grow-only scratch for the per-row records of sjd_verify, one buffer per
// (device, stream): calls on different streams never share records, and
// calls on one stream run in order, so a buffer replaced by a larger one is
// freed once its stream has drained the work that used it.
struct Scratch {
  std::mutex mu;
  std::map<std::pair<int, hipStream_t>, std::pair<void*, size_t>> buf;
};
Scratch g_scratch;

int scratch_get(hipStream_t stream, size_t bytes, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SJD_EHIP;
  std::lock_guard<std::mutex> lk(g_scratch.mu);
  auto& e = g_scratch.buf[std::make_pair(dev, stream)];
  if (e.second < bytes) {
    if (e.first) {
      // the previous buffer may still be in use by work queued on this stream
      if (hipStreamSynchronize(stream) != hipSuccess) return SJD_EHIP;
      (void)hipFree(e.first);
      e.first = nullptr;
      e.second = 0;
    }
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return SJD_ENOMEM;
    e.first = p;
    e.second = bytes;
  }
  *out = e.first;
  return SJD_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" const char* sjd_status_str(int s) {
  switch (s) {
    case SJD_OK: return "SJD_OK";
    case SJD_EINVAL: return "SJD_EINVAL: invalid argument";
    case SJD_ENOMEM: return "SJD_ENOMEM: device allocation failed";
    case SJD_EHIP: return "SJD_EHIP: HIP runtime error";
    case SJD_ESTATE: return "SJD_ESTATE: invalid context state";
    case SJD_ENOTSUP: return "SJD_ENOTSUP: not supported";
    case SJD_ENONFINITE: return "SJD_ENONFINITE: a logit is NaN or +inf";
    default: return "unknown sjd status";
  }
}

namespace sjd {
// The row kernel keeps one logits row in registers (V <= 65536) and the kept
// (top-k) tokens in LDS (at most kVerifyMaxK of them unless V is that small).
int check_verify_limits(int V, int top_k) {
  if (V > kVerifyMaxV) return SJD_ENOTSUP;
  const int k = (top_k <= 0 || top_k >= V) ? V : top_k;
  if (k > kVerifyMaxK) return SJD_ENOTSUP;
  return SJD_OK;
}

int check_verify_params(const sjd_verify_params* p) {
  if (!p) return SJD_EINVAL;
  if (p->B < 1 || p->B > 65535 || p->L < 1 || p->L > 64 || p->V < 4 || (p->V & 3) || p->V > (1 << 22))
    return SJD_EINVAL;
  if (p->K < 1 || p->K > 8 || p->D < 0 || (long)p->K * p->D > p->L) return SJD_EINVAL;
  if (p->top_k < 0 || !(p->temperature > 0.0f)) return SJD_EINVAL;
  if (p->flags & ~(SJD_AC | SJD_PD | SJD_CHECK_FINITE | SJD_FULL_SELECT)) return SJD_EINVAL;
  return check_verify_limits(p->V, p->top_k);
}
}  // namespace sjd

namespace {

// Argument checks shared by both verification entry points.
int check_verify_call(const sjd_verify_params* p, const sjd_verify_io* io) {
  int st = sjd::check_verify_params(p);
  if (st != SJD_OK) return st;
  if (!io || !io->d_cur || !io->d_draft || !io->d_draft_tok || !io->d_in_meta || !io->d_out_meta ||
      !io->d_out_tok || !io->d_out_next || (p->D * (p->K - 1) > 0 && !io->d_out_sib))
    return SJD_EINVAL;
  if (!aligned16(io->d_cur) || !aligned16(io->d_draft) || (io->d_dbg_p && !aligned16(io->d_dbg_p)))
    return SJD_EINVAL;
  return SJD_OK;
}

int enqueue_verify(const sjd_verify_params* p, const sjd_verify_io* io, int32_t* rec, hipStream_t stream) {
  sjd::VerifyArgs a{};
  a.B = p->B; a.L = p->L; a.V = p->V; a.K = p->K; a.D = p->D; a.top_k = p->top_k;
  a.T = p->temperature; a.flags = p->flags & (SJD_AC | SJD_PD); a.seed = p->seed; a.step = p->step;
  if (p->flags & SJD_FULL_SELECT) a.flags |= sjd::kFlagFullSelect;
  a.vis_lo = p->vis_lo; a.eol = p->eol_id; a.row_len = p->row_len;
  a.cur = io->d_cur; a.draft = io->d_draft; a.draft_bstride = (long long)p->L * p->V; a.q_off = nullptr;
  a.draft_tok = io->d_draft_tok; a.sib = io->d_sib; a.in_meta = io->d_in_meta;
  a.rec = rec; a.out_rows = io->d_out_rows; a.dbg_p = io->d_dbg_p;
  sjd::FinalizeOut o{};
  o.out_meta = io->d_out_meta; o.meta_stride = 8;
  o.out_tok = io->d_out_tok; o.tok_stride = p->L;
  o.out_next = io->d_out_next; o.next_stride = p->L;
  o.out_sib = io->d_out_sib; o.sib_stride = p->D * (p->K - 1);
  if (sjd::launch_verify(a, o, stream) != hipSuccess) return SJD_EHIP;
  return SJD_OK;
}

// SJD_CHECK_FINITE: counts NaN / +inf in both logits arrays into *cnt, then
// synchronises the stream; SJD_ENONFINITE if any was found.
int check_finite(const sjd_verify_params* p, const sjd_verify_io* io, int32_t* cnt, hipStream_t s) {
  const size_t n = (size_t)p->B * p->L * p->V;
  if (sjd::launch_count_nonfinite(io->d_cur, n, cnt, true, s) != hipSuccess ||
      sjd::launch_count_nonfinite(io->d_draft, n, cnt, false, s) != hipSuccess)
    return SJD_EHIP;
  int32_t h = 0;
  if (hipMemcpyAsync(&h, cnt, sizeof(int32_t), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return SJD_EHIP;
  return h ? SJD_ENONFINITE : SJD_OK;
}

}  // namespace

extern "C" int sjd_verify(const sjd_verify_params* p, const sjd_verify_io* io, void* stream) {
  int st = check_verify_call(p, io);
  if (st != SJD_OK) return st;
  void* rec = nullptr;
  const size_t rec_bytes = (size_t)p->B * p->L * sjd::kRecInts * sizeof(int32_t);
  st = scratch_get((hipStream_t)stream, rec_bytes + 256, &rec);
  if (st != SJD_OK) return st;
  if (p->flags & SJD_CHECK_FINITE) {
    st = check_finite(p, io, (int32_t*)((char*)rec + rec_bytes), (hipStream_t)stream);
    if (st != SJD_OK) return st;
  }
  return enqueue_verify(p, io, (int32_t*)rec, (hipStream_t)stream);
}

extern "C" int sjd_verify_noalloc(const sjd_verify_params* p, const sjd_verify_io* io, void* stream) {
  int st = check_verify_call(p, io);
  if (st != SJD_OK) return st;
  if ((long)p->B * p->L > SJD_VERIFY_NOALLOC_MAX_ROWS) return SJD_EINVAL;
  int32_t* rec = nullptr;
  if (sjd::noalloc_scratch(&rec) != hipSuccess) return SJD_EHIP;
  if (p->flags & SJD_CHECK_FINITE) {
    // the count word follows the largest record block
    st = check_finite(p, io, rec + (size_t)SJD_VERIFY_NOALLOC_MAX_ROWS * sjd::kRecInts, (hipStream_t)stream);
    if (st != SJD_OK) return st;
  }
  return enqueue_verify(p, io, rec, (hipStream_t)stream);
}
