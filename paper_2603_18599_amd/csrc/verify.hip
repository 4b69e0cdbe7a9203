// Verification of SJD-PAC windows (Alg. 1 of the paper): per-row kernel and
// per-trial finalize kernel.
//
// k_verify_rows: one 512-thread workgroup per (trial, row). The row's current
// logits (and draft logits, when the row has a draft distribution) are read
// once, coalesced as float4 per thread, and kept in registers for V <= 16384;
// larger vocabularies re-read the row from L2 in each pass. On chip the
// kernel finds the exact top-k threshold (radix select on order-preserving
// keys), the softmax statistics, the accept test(s), the residual draw,
// drafting candidates and the bonus draw, and writes one small record.
//
// k_verify_finalize: one wave per trial. Finds the first rejected spine row,
// the committed tokens, and assembles the next window.
//
// Arithmetic of every decision is fp32 with fp64 sums (the paper fixes no
// precision); contraction into FMA is off in this file so the rounding of
// each operation is the IEEE one.
#include "device.h"
#include "verify.h"

#pragma clang fp contract(off)

namespace sjd {

constexpr int kVB = 512;            // threads per row workgroup
constexpr int kVW = kVB / kWave;    // waves per row workgroup
constexpr uint64_t kNoKey = ~0ull;

struct VShared {
  uint32_t hist[2048];
  double red_d[kVW];
  uint64_t red_u[kVW];
  float red_f[kVW];
  int red_i[kVW];
  int bin, above;
};

// ------------------------------------------------------------ block helpers
SJD_DEV float block_max(float v, VShared& sh) {
  v = wave_max(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sh.red_f[w] = v;
  __syncthreads();
  float r = sh.red_f[0];
#pragma unroll
  for (int i = 1; i < kVW; ++i) r = fmaxf(r, sh.red_f[i]);
  __syncthreads();
  return r;
}
SJD_DEV double block_sum_d(double v, VShared& sh) {
  v = wave_sum_d(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sh.red_d[w] = v;
  __syncthreads();
  double r = 0.0;
#pragma unroll
  for (int i = 0; i < kVW; ++i) r += sh.red_d[i];
  __syncthreads();
  return r;
}
SJD_DEV uint64_t block_min_u64(uint64_t v, VShared& sh) {
  v = wave_min_u64(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sh.red_u[w] = v;
  __syncthreads();
  uint64_t r = sh.red_u[0];
#pragma unroll
  for (int i = 1; i < kVW; ++i) r = sh.red_u[i] < r ? sh.red_u[i] : r;
  __syncthreads();
  return r;
}
// exclusive prefix sum over the block (thread order)
SJD_DEV int block_excl_scan(int v, VShared& sh) {
  const int incl = wave_incl_scan(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == kWave - 1) sh.red_i[w] = incl;
  __syncthreads();
  int base = 0;
  for (int i = 0; i < w; ++i) base += sh.red_i[i];
  __syncthreads();
  return base + incl - v;
}

SJD_DEV float comp(const float4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; }
SJD_DEV float& comp(float4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; }

SJD_DEV uint64_t pack_key(float key, int x) {
  return ((uint64_t)__float_as_uint(key) << 32) | (uint32_t)x;
}

// ---------------------------------------------------------- row statistics
struct RowStats {
  float m;        // largest logit
  float T;
  uint32_t tau;   // key of the k-th largest logit
  int itau;       // largest index taken among logits equal to tau
  bool all;       // k >= V: every entry kept
  double invZ;    // 1 / sum of weights
  SJD_DEV bool in_set(float l, int x) const {
    if (all) return true;
    const uint32_t k = fkey(l);
    return k > tau || (k == tau && x <= itau);
  }
  SJD_DEV float prob(float l, int x) const {
    if (!in_set(l, x)) return 0.0f;
    const float w = expf((l - m) / T);
    return (float)((double)w * invZ);
  }
};

// Row data: NC > 0 keeps NC float4 chunks per thread in registers (chunk
// c = tid + i * kVB holds entries 4c .. 4c+3); NC == 0 re-reads global memory.
template <int NC>
struct Row {
  float4 v[NC];
  int nchunk;
  const float4* g;
  SJD_DEV static constexpr int count(int) { return NC; }
  SJD_DEV void load(const float* row, int V) {
    g = (const float4*)row;
    nchunk = V >> 2;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = threadIdx.x + i * kVB;
      v[i] = c < nchunk ? g[c] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
  }
  SJD_DEV float4 get(int i) const { return v[i]; }
};
template <>
struct Row<0> {
  int nchunk;
  const float4* g;
  SJD_DEV int count(int) const { return (nchunk + kVB - 1) / kVB; }
  SJD_DEV void load(const float* row, int V) {
    g = (const float4*)row;
    nchunk = V >> 2;
  }
  SJD_DEV float4 get(int i) const {
    const int c = threadIdx.x + i * kVB;
    return c < nchunk ? g[c] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  }
};

// Exact k-th largest under (value desc, index asc): radix select over the
// order-preserving keys (11 + 11 + 10 bits), then, if the threshold value is
// tied, over the indices of the tied entries (11 + 11 bits).
template <int NC>
SJD_DEV void topk_threshold(const Row<NC>& row, int V, int k, VShared& sh, RowStats& st) {
  st.all = (k <= 0 || k >= V);
  if (st.all) { st.tau = 0; st.itau = 0x7FFFFFFF; return; }
  const int tid = threadIdx.x;
  const int cnt = row.count(V);
  uint32_t prefix = 0, pmask = 0;
  int rem = k;
  int last_bin = 0;
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const int nb = pass == 2 ? 1024 : 2048;
    for (int b = tid; b < nb; b += kVB) sh.hist[b] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < cnt; ++i) {
      const int c = tid + i * kVB;
      if (c < row.nchunk) {
        const float4 v = row.get(i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t key = fkey(comp(v, e));
          if ((key & pmask) == prefix) atomicAdd(&sh.hist[(key >> shift) & (uint32_t)(nb - 1)], 1u);
        }
      }
    }
    __syncthreads();
    // bins in descending order: thread t owns reversed bins [t*per, t*per+per)
    const int per = nb / kVB;
    int cnts[4];
    int s = 0;
    for (int i = 0; i < per; ++i) {
      cnts[i] = (int)sh.hist[nb - 1 - (tid * per + i)];
      s += cnts[i];
    }
    int run = block_excl_scan(s, sh);
    for (int i = 0; i < per; ++i) {
      if (run < rem && run + cnts[i] >= rem) {
        sh.bin = nb - 1 - (tid * per + i);
        sh.above = run;
      }
      run += cnts[i];
    }
    __syncthreads();
    last_bin = sh.bin;
    const int above = sh.above;
    prefix |= (uint32_t)last_bin << shift;
    pmask |= (uint32_t)(nb - 1) << shift;
    rem -= above;
    __syncthreads();
  }
  st.tau = prefix;
  const int eq = (int)sh.hist[last_bin];
  __syncthreads();
  if (rem >= eq) {
    st.itau = 0x7FFFFFFF;
    return;
  }
  // rem-th smallest index among entries whose key equals tau
  uint32_t ipre = 0, imask = 0;
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 11 : 0;
    const int nb = 2048;
    for (int b = tid; b < nb; b += kVB) sh.hist[b] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < cnt; ++i) {
      const int c = tid + i * kVB;
      if (c < row.nchunk) {
        const float4 v = row.get(i);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t x = (uint32_t)(4 * c + e);
          if (fkey(comp(v, e)) == prefix && (x & imask) == ipre)
            atomicAdd(&sh.hist[(x >> shift) & 2047u], 1u);
        }
      }
    }
    __syncthreads();
    const int per = nb / kVB;
    int cnts[4];
    int s = 0;
    for (int i = 0; i < per; ++i) {
      cnts[i] = (int)sh.hist[tid * per + i];
      s += cnts[i];
    }
    int run = block_excl_scan(s, sh);
    for (int i = 0; i < per; ++i) {
      if (run < rem && run + cnts[i] >= rem) {
        sh.bin = tid * per + i;
        sh.above = run;
      }
      run += cnts[i];
    }
    __syncthreads();
    ipre |= (uint32_t)sh.bin << shift;
    imask |= 2047u << shift;
    rem -= sh.above;
    __syncthreads();
  }
  st.itau = (int)ipre;
}

template <int NC>
SJD_DEV void row_stats(Row<NC>& row, int V, int k, float T, VShared& sh, RowStats& st) {
  st.T = T;
  topk_threshold(row, V, k, sh, st);
  const int cnt = row.count(V);
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < cnt; ++i) {
    const float4 v = row.get(i);
    mx = fmaxf(mx, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
  }
  st.m = block_max(mx, sh);
  double z = 0.0;
#pragma unroll
  for (int i = 0; i < cnt; ++i) {
    const int c = threadIdx.x + i * kVB;
    if (c < row.nchunk) {
      const float4 v = row.get(i);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float l = comp(v, e);
        if (st.in_set(l, 4 * c + e)) z += (double)expf((l - st.m) / T);
      }
    }
  }
  st.invZ = 1.0 / block_sum_d(z, sh);
  if constexpr (NC > 0) {
    // keep probabilities instead of logits
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = threadIdx.x + i * kVB;
#pragma unroll
      for (int e = 0; e < 4; ++e) comp(row.v[i], e) = c < row.nchunk ? st.prob(comp(row.v[i], e), 4 * c + e) : 0.0f;
    }
  }
}

// probability of entry 4c+e given the chunk read from the row
template <int NC>
SJD_DEV float prob_of(const RowStats& st, const float4& v, int c, int e) {
  if constexpr (NC > 0) return comp(v, e);
  else return st.prob(comp(v, e), 4 * c + e);
}

// probability of one entry (any thread; reads global memory)
SJD_DEV float prob_scalar(const RowStats& st, const float* row, int x) {
  return st.prob(row[x], x);
}

struct Stages {
  int n;             // stages whose residual has been formed
  int cand[8];
  float Nf[8];       // normaliser of p^(s)
  float den[8];      // 1 - q mass of candidates rejected before stage s
  // rho^(n+1)(y): the unnormalised residual after n rejected stages. Loops
  // have fixed trip counts so every array index is a compile-time constant.
  SJD_DEV float rho(float py, float qy, int y) const {
    float r = py;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if (s < n) {
        bool ex = false;
#pragma unroll
        for (int t = 0; t < 8; ++t) ex |= (t < s) && (cand[t] == y);
        const float pk = r / Nf[s];
        const float qk = (ex || !(den[s] > 0.0f)) ? 0.0f : qy / den[s];
        const float d = pk - qk;
        r = d > 0.0f ? d : 0.0f;
      }
    }
    return r;
  }
};

// ------------------------------------------------------------ row kernel
template <int NC>
__global__ __launch_bounds__(kVB) void k_verify_rows(VerifyArgs a) {
  __shared__ VShared sh;
  const int j = blockIdx.x;
  const int b = blockIdx.y;
  const int L = a.L, V = a.V, K = a.K, Km1 = a.K - 1;
  const int32_t* meta = a.in_meta + 4 * (size_t)b;
  const int D_in = meta[0], n_q = meta[1];
  const long g0 = meta[2];
  const int n_s = L - Km1 * D_in;
  int32_t* rec = a.rec + ((size_t)b * L + j) * kRecInts;
  if (D_in < 0 || D_in > a.D || K * D_in > L || n_q < 0 || n_q > n_s) return;  // finalize flags the trial
  const bool ac = (a.flags & kFlagAC) != 0;
  const bool pd = (a.flags & kFlagPD) != 0 && Km1 > 0;
  auto forced = [&](long g) -> bool { return a.row_len > 0 && g >= 0 && (g % (a.row_len + 1)) == a.row_len; };

  // ---- classify the row (uniform over the block)
  bool spine = j < n_s;
  bool is_forced = false, need_p = true, has_q = false;
  int sib_d = -1, sib_k = 0, sib_tok = -1;
  if (spine) {
    is_forced = forced(g0 + j);
    has_q = !is_forced && j < n_q;
  } else {
    sib_d = (j - n_s) / Km1;
    sib_k = (j - n_s) % Km1 + 2;
    sib_tok = a.sib ? a.sib[((size_t)b * a.D + sib_d) * Km1 + (sib_k - 2)] : -1;
    is_forced = forced(g0 + sib_d + 1);
    if (sib_tok < 0 || forced(g0 + sib_d)) need_p = false;
    else if (is_forced) need_p = false;
  }
  if (is_forced && spine) need_p = false;
  if (a.dbg_p) need_p = true;

  const float* cur_row = a.cur + ((size_t)b * L + j) * V;
  Row<NC> P;
  RowStats ps{};
  if (need_p) {
    P.load(cur_row, V);
    row_stats(P, V, a.top_k, a.T, sh, ps);
    if (a.dbg_p) {
      float4* dst = (float4*)(a.dbg_p + ((size_t)b * L + j) * V);
      const int cnt = P.count(V);
#pragma unroll
      for (int i = 0; i < cnt; ++i) {
        const int c = threadIdx.x + i * kVB;
        if (c < P.nchunk) {
          const float4 v = P.get(i);
          float4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) comp(o, e) = prob_of<NC>(ps, v, c, e);
          dst[c] = o;
        }
      }
    }
  }

  // ---- sibling rows: bonus draw from the sibling's own output row
  if (!spine) {
    int tok = -1, stage = 0;
    if (sib_tok < 0 || forced(g0 + sib_d)) {
      tok = -1; stage = 0;
    } else if (is_forced) {
      tok = -1; stage = -1;
    } else {
      const Stream rs(a.seed, kTagBonus, 0, (uint32_t)j, (uint32_t)b, a.step);
      uint64_t best = kNoKey;
      const int cnt = P.count(V);
#pragma unroll
      for (int i = 0; i < cnt; ++i) {
        const int c = threadIdx.x + i * kVB;
        if (c < P.nchunk) {
          const float4 v = P.get(i);
          const uint4 w = rs.block((uint32_t)c);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float pw = prob_of<NC>(ps, v, c, e);
            if (pw > 0.0f) {
              const uint32_t wd = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
              const uint64_t pk = pack_key(exp1(wd) / pw, 4 * c + e);
              best = pk < best ? pk : best;
            }
          }
        }
      }
      best = block_min_u64(best, sh);
      tok = best == kNoKey ? -1 : (int)(uint32_t)best;
    }
    if (threadIdx.x == 0) {
      rec[0] = tok; rec[1] = stage;
      for (int t = 0; t < 7; ++t) rec[2 + t] = -1;
      rec[9] = tok;
      if (a.out_rows) {
        int32_t* o = a.out_rows + ((size_t)b * L + j) * 2;
        o[0] = stage == -1 ? a.eol : (tok < 0 ? -1 : tok + a.vis_lo);
        o[1] = stage;
      }
    }
    return;
  }

  // ---- spine rows
  if (is_forced) {
    if (threadIdx.x == 0) {
      rec[0] = -1; rec[1] = -1;
      for (int t = 0; t < 7; ++t) rec[2 + t] = -1;
      rec[9] = -1;
      if (a.out_rows) {
        int32_t* o = a.out_rows + ((size_t)b * L + j) * 2;
        o[0] = a.eol; o[1] = -1;
      }
    }
    return;
  }

  // candidates: the spine draft, then (tree rows) its siblings; an
  // out-of-range or repeated candidate ends the list
  Stages stg;
  stg.n = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) { stg.cand[t] = -1; stg.Nf[t] = 1.0f; stg.den[t] = 1.0f; }
  int ncand = 0;
  if (has_q) {
    const int x0 = a.draft_tok[(size_t)b * L + j] - a.vis_lo;
    if (x0 >= 0 && x0 < V) {
      stg.cand[0] = x0;
      ncand = 1;
      if (j < D_in && a.sib) {
        bool open = true;
#pragma unroll
        for (int k = 0; k < 7; ++k) {
          if (open && k < Km1) {
            int y = a.sib[((size_t)b * a.D + j) * Km1 + k];
            bool stop = y < 0;
            y -= a.vis_lo;
            stop |= (y < 0 || y >= V);
#pragma unroll
            for (int t = 0; t < 8; ++t) stop |= (t <= k) && (stg.cand[t] == y);
            if (stop) open = false;
            else { stg.cand[k + 1] = y; ncand = k + 2; }
          }
        }
      }
    }
  }

  int out_tok = -1, out_stage = 0;
  if (ncand > 0) {
    const size_t qrow = (size_t)b * a.draft_bstride + (size_t)((a.q_off ? a.q_off[b] : 0) + j) * V;
    const float* draft_row = a.draft + qrow;
    Row<NC> Q;
    RowStats qs{};
    Q.load(draft_row, V);
    row_stats(Q, V, a.top_k, a.T, sh, qs);

    float Qsum = 0.0f;
    float Nf = 1.0f;
    bool done = false;
    for (int k = 1; k <= ncand && !done; ++k) {
      int x = stg.cand[0];
#pragma unroll
      for (int t = 1; t < 8; ++t) x = (t == k - 1) ? stg.cand[t] : x;
      const float den = 1.0f - Qsum;
      const float px = prob_scalar(ps, cur_row, x);
      const float qx = prob_scalar(qs, draft_row, x);
      const float pk = stg.rho(px, qx, x) / Nf;
      const float qk = den > 0.0f ? qx / den : 0.0f;
      const Stream us(a.seed, kTagAcc, (uint32_t)(k - 1), (uint32_t)j, (uint32_t)b, a.step);
      const float u = u01(us.word(0));
      const bool acc = qk > 0.0f ? (u < pk / qk) : (pk > 0.0f);
      if (acc) {
        out_tok = x;
        out_stage = k;
        done = true;
        break;
      }
      // residual of this stage
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (t == stg.n) { stg.Nf[t] = Nf; stg.den[t] = den; }
      stg.n += 1;
      double nd = 0.0;
      const int cnt = P.count(V);
#pragma unroll
      for (int i = 0; i < cnt; ++i) {
        const int c = threadIdx.x + i * kVB;
        if (c < P.nchunk) {
          const float4 pv = P.get(i), qv = Q.get(i);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            nd += (double)stg.rho(prob_of<NC>(ps, pv, c, e), prob_of<NC>(qs, qv, c, e), 4 * c + e);
        }
      }
      nd = block_sum_d(nd, sh);
      Qsum = Qsum + qx;
      if (!(nd > 0.0)) {
        stg.n -= 1;  // no residual mass: draw from p^(k) itself
        break;
      }
      Nf = (float)nd;
    }
    // draw from the last residual (stage number = candidates tried)
    if (out_stage == 0) {
      // candidates tried: all of them unless the loop left through the
      // zero-mass exit, in which case that stage was tried too
      const int tried = stg.n + (stg.n < ncand ? 1 : 0);
      const Stream rs(a.seed, kTagRes, (uint32_t)tried, (uint32_t)j, (uint32_t)b, a.step);
      uint64_t best = kNoKey;
      const int cnt = P.count(V);
#pragma unroll
      for (int i = 0; i < cnt; ++i) {
        const int c = threadIdx.x + i * kVB;
        if (c < P.nchunk) {
          const float4 pv = P.get(i), qv = Q.get(i);
          const uint4 w = rs.block((uint32_t)c);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float r = stg.rho(prob_of<NC>(ps, pv, c, e), prob_of<NC>(qs, qv, c, e), 4 * c + e);
            if (r > 0.0f) {
              const uint32_t wd = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
              const uint64_t pk = pack_key(exp1(wd) / r, 4 * c + e);
              best = pk < best ? pk : best;
            }
          }
        }
      }
      best = block_min_u64(best, sh);
      out_tok = best == kNoKey ? -1 : (int)(uint32_t)best;
    }
  } else {
    // no draft distribution (appended placeholder) or no valid candidate:
    // a plain draw from p, counted as a rejection
    const Stream rs(a.seed, kTagRes, 0, (uint32_t)j, (uint32_t)b, a.step);
    uint64_t best = kNoKey;
    const int cnt = P.count(V);
#pragma unroll
    for (int i = 0; i < cnt; ++i) {
      const int c = threadIdx.x + i * kVB;
      if (c < P.nchunk) {
        const float4 v = P.get(i);
        const uint4 w = rs.block((uint32_t)c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pw = prob_of<NC>(ps, v, c, e);
          if (pw > 0.0f) {
            const uint32_t wd = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
            const uint64_t pk = pack_key(exp1(wd) / pw, 4 * c + e);
            best = pk < best ? pk : best;
          }
        }
      }
    }
    best = block_min_u64(best, sh);
    out_tok = best == kNoKey ? -1 : (int)(uint32_t)best;
    out_stage = 0;
  }

  // vanilla SJD: a fresh draw from p replaces the row in the next window
  int fresh = out_tok;
  if (!ac) {
    const Stream rs(a.seed, kTagFresh, 0, (uint32_t)j, (uint32_t)b, a.step);
    uint64_t best = kNoKey;
    const int cnt = P.count(V);
#pragma unroll
    for (int i = 0; i < cnt; ++i) {
      const int c = threadIdx.x + i * kVB;
      if (c < P.nchunk) {
        const float4 v = P.get(i);
        const uint4 w = rs.block((uint32_t)c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pw = prob_of<NC>(ps, v, c, e);
          if (pw > 0.0f) {
            const uint32_t wd = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
            const uint64_t pk = pack_key(exp1(wd) / pw, 4 * c + e);
            best = pk < best ? pk : best;
          }
        }
      }
    }
    best = block_min_u64(best, sh);
    fresh = best == kNoKey ? -1 : (int)(uint32_t)best;
  }

  // proactive drafting: K-1 draws without replacement from p, excluding the
  // token this row carries into the next window
  int pds[7] = {-1, -1, -1, -1, -1, -1, -1};
  if (pd) {
    const int excl = ac ? out_tok : fresh;
    const Stream rs(a.seed, kTagPd, 0, (uint32_t)j, (uint32_t)b, a.step);
    uint64_t loc[7];
#pragma unroll
    for (int t = 0; t < 7; ++t) loc[t] = kNoKey;
    const int cnt = P.count(V);
#pragma unroll
    for (int i = 0; i < cnt; ++i) {
      const int c = threadIdx.x + i * kVB;
      if (c < P.nchunk) {
        const float4 v = P.get(i);
        const uint4 w = rs.block((uint32_t)c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int x = 4 * c + e;
          const float pw = prob_of<NC>(ps, v, c, e);
          if (pw > 0.0f && x != excl) {
            const uint32_t wd = e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
            uint64_t pk = pack_key(exp1(wd) / pw, x);
            // insert into the thread's ascending list of the Km1 smallest
#pragma unroll
            for (int t = 0; t < 7; ++t) {
              if (t < Km1 && pk < loc[t]) {
                const uint64_t tmp = loc[t];
                loc[t] = pk;
                pk = tmp;
              }
            }
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < 7; ++t) {
      if (t < Km1) {
        const uint64_t best = block_min_u64(loc[0], sh);
        if (best != kNoKey) {
          pds[t] = (int)(uint32_t)best;
          if (loc[0] == best) {
#pragma unroll
            for (int u = 0; u < 6; ++u) loc[u] = loc[u + 1];
            loc[6] = kNoKey;
          }
        }
      }
    }
  }

  if (threadIdx.x == 0) {
    rec[0] = out_tok;
    rec[1] = out_stage;
    for (int t = 0; t < 7; ++t) rec[2 + t] = pds[t];
    rec[9] = fresh;
    if (a.out_rows) {
      int32_t* o = a.out_rows + ((size_t)b * L + j) * 2;
      o[0] = out_tok < 0 ? -1 : out_tok + a.vis_lo;
      o[1] = out_stage;
    }
  }
}

// ------------------------------------------------------------ finalize
__global__ __launch_bounds__(kWave) void k_verify_finalize(VerifyArgs a, FinalizeOut o) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int L = a.L, V = a.V, K = a.K, Km1 = a.K - 1, D = a.D;
  const int32_t* meta = a.in_meta + 4 * (size_t)b;
  const int D_in = meta[0];
  const long g0 = meta[2];
  const int n_s = L - Km1 * D_in;
  const int32_t* rec = a.rec + (size_t)b * L * kRecInts;
  if (D_in < 0 || D_in > D || K * D_in > L || meta[1] < 0 || meta[1] > n_s) {
    // invalid window description: the trial is marked and nothing else written
    if (lane == 0) {
      int32_t* om = o.out_meta + (size_t)b * o.meta_stride;
      om[0] = -1; om[1] = -1; om[2] = 0; om[3] = 0; om[4] = 0; om[5] = 0; om[6] = 0; om[7] = 0;
    }
    return;
  }
  const bool ac = (a.flags & kFlagAC) != 0;
  const bool pd = (a.flags & kFlagPD) != 0 && Km1 > 0;
  auto forced = [&](long g) -> bool { return a.row_len > 0 && g >= 0 && (g % (a.row_len + 1)) == a.row_len; };
  auto tokof = [&](int r) -> int { return rec[r * kRecInts + 1] == -1 ? a.eol : rec[r * kRecInts] + a.vis_lo; };

  // first spine row whose own draft was not accepted
  const bool rej = lane < n_s && !(rec[lane * kRecInts + 1] == -1 || rec[lane * kRecInts + 1] == 1);
  const uint64_t bal = __ballot(rej);
  const int r = bal ? (int)__ffsll((unsigned long long)bal) - 1 : -1;

  int n_c, acc_k = 0;
  int32_t* otok = o.out_tok + (size_t)b * o.tok_stride;
  if (r < 0) {
    n_c = n_s;
  } else if (rec[r * kRecInts + 1] >= 2) {
    acc_k = rec[r * kRecInts + 1];
    n_c = r + 2;
  } else {
    n_c = r + 1;
  }
  if (lane < L) {
    int t = -1;
    if (lane < n_c) {
      if (acc_k >= 2 && lane == r) t = rec[r * kRecInts] + a.vis_lo;
      else if (acc_k >= 2 && lane == r + 1) t = tokof(n_s + r * Km1 + (acc_k - 2));
      else t = tokof(lane);
    }
    otok[lane] = t;
  }

  int Dn = 0;
  if (pd && r >= 0) {
    Dn = D;
    if (n_s - n_c < Dn) Dn = n_s - n_c;
    if (L / K < Dn) Dn = L / K;
    if (Dn < 0) Dn = 0;
  }
  const int n_s2 = L - Km1 * Dn;
  int n_q2 = n_s - n_c;
  if (n_q2 < 0) n_q2 = 0;
  if (n_q2 > n_s2) n_q2 = n_s2;

  int32_t* onext = o.out_next + (size_t)b * o.next_stride;
  if (lane < L) {
    int t = -1;
    if (lane < n_s2) {
      const int jj = n_c + lane;
      const long g = g0 + n_c + lane;
      if (jj < n_s) {
        if (rec[jj * kRecInts + 1] == -1) t = a.eol;
        else t = (ac ? rec[jj * kRecInts] : rec[jj * kRecInts + 9]) + a.vis_lo;
      } else if (forced(g)) {
        t = a.eol;
      } else {
        const Stream is(a.seed, kTagInit, 0, (uint32_t)lane, (uint32_t)b, a.step);
        const uint32_t w = is.word(0);
        t = a.vis_lo + (int)(((uint64_t)w * (uint64_t)V) >> 32);
      }
    }
    onext[lane] = t;
  }
  int32_t* osib = o.out_sib + (size_t)b * o.sib_stride;
  for (int i = lane; i < D * Km1; i += kWave) {
    const int d = i / Km1, k = i % Km1;
    int t = -1;
    if (d < Dn) {
      const int jj = n_c + d;
      if (rec[jj * kRecInts + 1] != -1) {
        const int y = rec[jj * kRecInts + 2 + k];
        t = y < 0 ? -1 : y + a.vis_lo;
      }
    }
    osib[i] = t;
  }
  if (lane == 0) {
    int32_t* om = o.out_meta + (size_t)b * o.meta_stride;
    om[0] = n_c; om[1] = r; om[2] = Dn; om[3] = n_s2; om[4] = n_q2; om[5] = acc_k;
    om[6] = (int32_t)(g0 + n_c); om[7] = 0;
  }
}

// ------------------------------------------------------------ launch
hipError_t launch_verify(const VerifyArgs& a, const FinalizeOut& o, hipStream_t s) {
  const dim3 grid(a.L, a.B);
  const int nchunk = a.V / 4;
  if (nchunk <= kVB) hipLaunchKernelGGL(k_verify_rows<1>, grid, dim3(kVB), 0, s, a);
  else if (nchunk <= 2 * kVB) hipLaunchKernelGGL(k_verify_rows<2>, grid, dim3(kVB), 0, s, a);
  else if (nchunk <= 4 * kVB) hipLaunchKernelGGL(k_verify_rows<4>, grid, dim3(kVB), 0, s, a);
  else if (nchunk <= 8 * kVB) hipLaunchKernelGGL(k_verify_rows<8>, grid, dim3(kVB), 0, s, a);
  else hipLaunchKernelGGL(k_verify_rows<0>, grid, dim3(kVB), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_verify_finalize, dim3(a.B), dim3(kWave), 0, s, a, o);
  return hipGetLastError();
}

}  // namespace sjd
