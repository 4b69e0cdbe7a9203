// Step bookkeeping kernels: window layout from the device state, prefill
// windows, state initialisation, KV commit (moving an accepted sibling's
// key/value row) and the state update after verification. Everything stays
// in device memory; the host only enqueues.
//
// Window layout (the paper fixes L verified positions per forward, Sec. 3.3,
// and K candidates at each of the first D positions after a rejection,
// Sec. 4.1): slot 0 holds the pending token (last committed, not yet cached)
// at position n; slot i, 1 <= i < n_s, holds spine draft i-1 at n + i;
// slot n_s + d(K-1) + k-2 holds sibling k of depth d at n + 1 + d and sees
// slots 0..d and itself. A missing sibling slot is fed token vis_lo.
#include "device.h"
#include "forward.h"
#include "step.h"

namespace sjd {

__global__ void k_build_window(const DevState* st, Window* w, int L, int K, int vis_lo, Streams sm) {
  const int a = threadIdx.x;
  const bool multi = sm.mode != kStreamsOne;
  const int z = multi ? a >> 5 : 0;      // stream of this row
  const int loc = multi ? (a & 31) : a;  // window row within its stream
  if (loc >= L) {  // padding row of a multi-stream window: never read, never cached
    if (multi) {
      w->tok[a] = vis_lo;
      w->pos[a] = st->n;
      w->anc[a] = 0ull;
    }
    return;
  }
  // batched: stream z is image z; guided: streams 2b, 2b + 1 are image b
  const DevState* d = multi ? st + stream_image(sm, z) : st;
  const bool unc = multi && stream_uncond(sm, z);
  const int n = d->n, n_s = d->n_s;
  int tok, pos;
  uint64_t anc;
  if (loc < n_s) {
    tok = loc == 0 ? (unc ? d->pending_u : d->pending) : d->spine[loc - 1];
    pos = n + loc;
    anc = loc == 63 ? ~0ull : ((1ull << (loc + 1)) - 1ull);
  } else {
    const int t = loc - n_s, dd = t / (K - 1), k = t % (K - 1);
    const int y = d->sib[dd * (K - 1) + k];
    tok = y >= 0 ? y : vis_lo;
    pos = n + 1 + dd;
    anc = ((1ull << (dd + 1)) - 1ull) | (1ull << loc);
  }
  w->tok[a] = tok;
  w->pos[a] = unc ? pos + d->delta_u : pos;
  w->anc[a] = anc;
}

__global__ void k_build_prefill(const int32_t* prompt, int start, int M, Window* w) {
  const int a = threadIdx.x;
  if (a >= M) return;
  w->tok[a] = prompt[start + a];
  w->pos[a] = start + a;
  w->anc[a] = a == 63 ? ~0ull : ((1ull << (a + 1)) - 1ull);
}

// Placeholders of the first window: uniform over the support (stream tag 6,
// trial 0, step word 0xFFFFFFFF, row = window index), the row end token at
// forced positions; no draft distributions, no siblings.
__global__ void k_state_init(DevState* st, const int32_t* prompt, int n_p, const int32_t* uncond, int n_u, int L,
                             int V, int vis_lo, int eol, int row_len, uint64_t seed) {
  const int i = threadIdx.x;
  if (i == 0) {
    st->n = n_p - 1;
    st->pending = prompt[n_p - 1];
    st->pending_u = uncond ? uncond[n_u - 1] : prompt[n_p - 1];
    st->delta_u = uncond ? n_u - n_p : 0;
    st->pad2[0] = st->pad2[1] = 0;
    st->n_s = L;
    st->D_in = 0;
    st->n_q = 0;
    st->g0 = 0;
    st->q_off = 0;
    st->pad = 0;
    for (int t = 0; t < 8; ++t) st->meta[t] = 0;
  }
  if (i < 64) {
    st->sib[i] = -1;
    st->tok[i] = -1;
    int t = -1;
    if (i < L) {
      const bool forced = row_len > 0 && (i % (row_len + 1)) == row_len;
      if (forced) {
        t = eol;
      } else {
        const Stream is(seed, kTagInit, 0, (uint32_t)i, 0u, 0xFFFFFFFFu);
        t = vis_lo + (int)(((uint64_t)is.word(0) * (uint64_t)V) >> 32);
      }
    }
    st->spine[i] = t;
  }
}

// Accepted sibling (meta[5] = k >= 2 at first rejected row r): its key and
// value move from cache position n + n_s + r(K-1) + k-2 to n + r + 1.
// grid (layers, Hkv, caches), block hd: cache z is the one at c + z *
// sstride; without guidance it is image z's, with guidance caches 2b and
// 2b + 1 are image b's text and unconditional streams (the latter's
// positions shifted by the image's delta_u).
__global__ void k_kv_move(const DevState* st, KvPlanes c, int Hkv, int hd, int cap, int K, int guided) {
  const int z = blockIdx.z;
  st += guided ? z >> 1 : z;
  const int off = guided && (z & 1) ? st->delta_u : 0;
  c.kc += z * c.sstride;
  c.kc_lo += z * c.sstride;
  c.vt += z * c.sstride;
  c.vt_lo += z * c.sstride;
  const int acc_k = st->meta[5];
  if (acc_k < 2) return;
  const int r = st->meta[1];
  const int src = st->n + off + st->n_s + r * (K - 1) + (acc_k - 2);
  const int dst = st->n + off + r + 1;
  const int l = blockIdx.x, kh = blockIdx.y, j = threadIdx.x;
  const size_t base = ((size_t)l * Hkv + kh) * cap * hd;
  const size_t ks = base + kv_key_off(src, j, hd), kd = base + kv_key_off(dst, j, hd);
  const size_t vs = base + kv_val_off(src, j, hd), vd = base + kv_val_off(dst, j, hd);
  c.kc[kd] = c.kc[ks];
  c.kc_lo[kd] = c.kc_lo[ks];
  c.vt[vd] = c.vt[vs];
  c.vt_lo[vd] = c.vt_lo[vs];
}

// grid B (one block per image of a batch); host_n[b] (pinned host memory)
// receives the image's cached rows after the step
__global__ void k_state_update(DevState* st, int32_t* out_meta, int32_t* out_tok, int32_t* out_next, int L,
                               int32_t* host_n) {
  __shared__ int32_t sm[8];
  const int i = threadIdx.x, b = blockIdx.x;
  st += b;
  if (out_meta) out_meta += 8 * b;
  if (out_tok) out_tok += L * b;
  if (out_next) out_next += L * b;
  if (i < 8) sm[i] = st->meta[i];
  __syncthreads();
  const int n_c = sm[0];
  const int n_new = st->n + (n_c > 0 ? n_c : 0);
  if (out_tok && i < L) out_tok[i] = st->tok[i];
  if (out_next && i < L) out_next[i] = st->spine[i];
  if (out_meta && i < 8) out_meta[i] = i == 7 ? n_new : sm[i];
  if (host_n && i == 0) host_n[b] = n_new;
  __syncthreads();
  if (i == 0 && n_c > 0) {
    st->pending = st->tok[n_c - 1];
    st->pending_u = st->tok[n_c - 1];
    st->n = n_new;
    st->n_s = sm[3];
    st->D_in = sm[2];
    st->n_q = sm[4];
    st->g0 = sm[6];
    st->q_off = n_c;
    st->meta[7] = n_new;
  }
}

// Caller-supplied drafts of the next step: a plain chain (no drafting
// siblings) whose row j carries tok[j]; with has_q, row j's draft
// distribution is row j of the draft logits (q_off 0), otherwise no row has
// one and every row draws from its own distribution.
__global__ void k_set_drafts(DevState* st, const int32_t* tok, int L, int has_q) {
  const int j = threadIdx.x;
  if (j < L) st->spine[j] = tok[j];
  if (j == 0) {
    st->n_s = L;
    st->D_in = 0;
    st->n_q = has_q ? L : 0;
    st->q_off = 0;
  }
}

// SJD_CHECK_FINITE: counts the NaN and +inf entries of p[0 .. n) into *cnt
// (-inf marks an excluded token and is allowed).
__global__ void k_zero1(int32_t* cnt) { *cnt = 0; }
__global__ __launch_bounds__(256) void k_count_nonfinite(const float* p, size_t n, int32_t* cnt) {
  int bad = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const float v = p[i];
    bad += (v != v) || (v == INFINITY);
  }
  const int tot = wave_sum_i(bad);
  if ((threadIdx.x & (kWave - 1)) == 0 && tot) atomicAdd(cnt, tot);
}

hipError_t launch_count_nonfinite(const float* p, size_t n, int32_t* cnt, bool reset, hipStream_t s) {
  if (reset) hipLaunchKernelGGL(k_zero1, dim3(1), dim3(1), 0, s, cnt);
  if (n > 0) {
    size_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(k_count_nonfinite, dim3((unsigned)blocks), dim3(256), 0, s, p, n, cnt);
  }
  return hipGetLastError();
}

hipError_t launch_set_drafts(DevState* st, const int32_t* tok, int L, bool has_q, hipStream_t s) {
  if (L < 1 || L > 64) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_set_drafts, dim3(1), dim3(64), 0, s, st, tok, L, has_q ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_build_window(const DevState* st, Window* w, int L, int K, int vis_lo, const Streams& sm,
                               hipStream_t s) {
  const bool multi = sm.mode != kStreamsOne;
  if (multi && (sm.nz < 1 || sm.nz > kMaxStreams || L > 32)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_build_window, dim3(1), dim3(multi ? 32 * sm.nz : 64), 0, s, st, w, L, K, vis_lo, sm);
  return hipGetLastError();
}
hipError_t launch_build_prefill(const int32_t* prompt, int start, int M, Window* w, hipStream_t s) {
  hipLaunchKernelGGL(k_build_prefill, dim3(1), dim3(64), 0, s, prompt, start, M, w);
  return hipGetLastError();
}
hipError_t launch_state_init(DevState* st, const int32_t* prompt, int n_p, const int32_t* uncond, int n_u, int L,
                             int V, int vis_lo, int eol, int row_len, uint64_t seed, hipStream_t s) {
  hipLaunchKernelGGL(k_state_init, dim3(1), dim3(64), 0, s, st, prompt, n_p, uncond, n_u, L, V, vis_lo, eol, row_len,
                     seed);
  return hipGetLastError();
}
hipError_t launch_kv_move(const DevState* st, const KvPlanes& c, int layers, int Hkv, int hd, int cap, int K,
                          int ncache, bool guided, hipStream_t s) {
  hipLaunchKernelGGL(k_kv_move, dim3(layers, Hkv, ncache), dim3(hd), 0, s, st, c, Hkv, hd, cap, K, guided ? 1 : 0);
  return hipGetLastError();
}
hipError_t launch_state_update(DevState* st, int32_t* out_meta, int32_t* out_tok, int32_t* out_next, int L, int B,
                               int32_t* host_n, hipStream_t s) {
  hipLaunchKernelGGL(k_state_update, dim3(B), dim3(64), 0, s, st, out_meta, out_tok, out_next, L, host_n);
  return hipGetLastError();
}

}  // namespace sjd
