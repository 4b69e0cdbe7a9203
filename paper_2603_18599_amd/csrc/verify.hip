// Verification of SJD-PAC windows (Alg. 1 of the paper): per-row kernel and
// per-trial finalize kernel.
//
// k_verify_rows: one workgroup per (trial, row). The row is read once,
// coalesced (float4 per thread), into registers. Every full-row pass is kept
// to a few instructions per logit; the exponentials, normalisers and all
// decisions run over the compact list of kept tokens (at most 2048):
//  - top-k selection: one histogram over bins of the row's [min, max] range
//    (well spread for real logits, so the LDS atomics rarely collide); one
//    pass then marks every entry of a bin above the threshold bin in a
//    bitmap of the kept set and collects the threshold bin's entries, whose
//    exact (value desc, index asc) rank decides which of them join it; a
//    radix select over order-preserving keys is the fallback for degenerate
//    rows (many equal values);
//  - compaction: per-word prefix popcounts of the bitmap give each kept token
//    its rank, which indexes the compact arrays and the random stream (four
//    consecutive ranks share one Philox block);
//  - the draft row (when the row has a draft distribution) goes through the
//    same selection into a second bitmap; one pass stores its logits at the
//    target's kept entries and at its own kept entries (for its normaliser);
//  - accept tests, residual draws (Theorem 2's recursion for several
//    candidates), drafting candidates and bonus draws run over the compact
//    list only.
// k_verify_finalize: one wave per trial. Finds the first rejected spine row,
// the committed tokens, and assembles the next window.
//
// Every decision is taken in fp32 with fp64 sums (the paper fixes no
// precision); contraction into FMA is off in this file so each operation
// rounds as IEEE specifies.
#include <mutex>
#include <type_traits>
#include <vector>

#include "device.h"
#include "sjd.h"
#include "verify.h"

#pragma clang fp contract(off)

namespace sjd {

// per-trial stride of a verify input whose packed per-trial size is `packed`
SJD_DEV size_t trial_stride(const VerifyArgs& a, size_t packed) {
  return a.state_stride > 0 ? (size_t)a.state_stride : packed;
}

constexpr uint64_t kNoKey = ~0ull;
constexpr int kKcap = kVerifyMaxK;   // kept tokens per row held on chip
constexpr int kCandCap = 256;        // threshold-bin entries ranked exactly
constexpr int kBins = 2048;

constexpr int kFastBins = 1024;  // candidate-path threshold histogram (bins over [lo, max])
constexpr int kSampBins = 512;   // candidate-path sample histogram (bins over the sample range)

// Compact list of a row's kept tokens, by rank (index order).
struct SpList {
  uint16_t x[kKcap];  // token index,
  float p[kKcap];     //   target probability,
  float q[kKcap];     //   draft probability
};

template <int BLOCK, int NC>
struct VSh {
  static constexpr int W = BLOCK / kWave;
  static constexpr int NW = BLOCK * NC / 8;  // bitmap words (32 entries each)
  // candidate path: entries of a row at or above its estimated threshold,
  // CAPW per wave
  static constexpr int CAP = BLOCK >= 1024 ? 4096 : 3072;
  static constexpr int CAPW = CAP / W;
  static_assert(W <= 16, "the drafting merge holds 8 keys of each wave in two registers per lane");
  // scratch of the full-row selection (the fallback path)
  struct OldSel {
    uint32_t bmq[NW];   // kept set of the draft row
    int32_t preq[NW];   // its per-word prefix popcounts
    union {
      uint32_t hist[kBins];
      float qc[kKcap];  // draft row's kept weights (its normaliser)
    };
    uint32_t hist_q[kBins];  // the draft row's histogram when both rows are selected together
    // per selected row (target, draft): threshold-bin entries, then sentinels
    // that outrank nothing (-inf, INT_MAX)
    float cand_v[2][kCandCap + 8];
    int cand_x[2][kCandCap + 8];
  };
  // scratch of the candidate path
  struct FastSel {
    float cv[CAP];    // target candidates: logit (after the normaliser: weight, or -1 if not kept)
    float cq[CAP];    //   the draft logit of the same token
    int32_t cx[CAP];  //   token index
    uint32_t hist[2][kFastBins];
    float tb_v[2][kCandCap + 8];  // threshold-bin entries, then sentinels
    int tb_x[2][kCandCap + 8];
    int tb_s[1][kCandCap + 8];  // the target's threshold-bin entries' candidate slots
  };
  uint32_t bm[NW];    // kept set of the target row
  int32_t pre[NW];    // its per-word prefix popcounts
  union {
    SpList sp;        // compact list of the target row's kept tokens
    float dv[CAP];    // candidate path: the draft row's candidates (dead before the list is built)
  } u;
  union {
    OldSel o;
    FastSel f;
  };
  uint64_t pd_w[W * 8];  // per-wave drafting keys
  int pd_o[8];            // the drafting draws
  double red_d[2 * W];
  uint64_t red_u[W];
  alignas(16) float red_f[8 * W];
  int red_i[2 * W];
  float tau_v[2];
  int tau_x[2], bin[2], above[2], ncand[2];
  int wcnt[2][W];  // candidate path: candidates per wave (-1: overflow)
  int fflag;       // candidate path: a row needs the full selection
};
static_assert(kBins == kKcap, "the draft weights reuse the histogram");

// ------------------------------------------------------------ block helpers
template <int W>
SJD_DEV void block_maxmin(float& mx, float& mn, float* red) {
  mx = wave_max_dpp(mx);
  mn = -wave_max_dpp(-mn);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) {
    red[w] = mx;
    red[W + w] = mn;
  }
  __syncthreads();
  mx = red[0];
  mn = red[W];
#pragma unroll
  for (int i = 1; i < W; ++i) {
    mx = fmaxf(mx, red[i]);
    mn = fminf(mn, red[W + i]);
  }
  __syncthreads();
}
template <int W>
SJD_DEV double block_sum_d(double v, double* red) {
  v = wave_sum_d_dpp(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  double r = 0.0;
#pragma unroll
  for (int i = 0; i < W; ++i) r += red[i];
  __syncthreads();
  return r;
}
template <int W>
SJD_DEV uint64_t block_min_u64(uint64_t v, uint64_t* red) {
  v = wave_min_u64_dpp(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) red[w] = v;
  __syncthreads();
  uint64_t r = red[0];
#pragma unroll
  for (int i = 1; i < W; ++i) r = red[i] < r ? red[i] : r;
  __syncthreads();
  return r;
}
// exclusive prefix sum over the block (thread order)
template <int W>
SJD_DEV int block_excl_scan(int v, int* red) {
  const int incl = wave_incl_scan_dpp(v);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == kWave - 1) red[w] = incl;
  __syncthreads();
  int base = 0;
  for (int i = 0; i < w; ++i) base += red[i];
  __syncthreads();
  return base + incl - v;
}

// Max / min that propagate NaN (IEEE 754-2019 maximum / minimum): one
// v_maximum3 / v_minimum3 per pair, with no quieting copy of each operand
// (fmaxf / fminf make one, which doubles the live registers of a pass over
// a row held in registers). Logits are finite or -inf here.
SJD_DEV float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }
SJD_DEV float vmin(float a, float b) { return __builtin_elementwise_minimum(a, b); }

// d / T with the division skipped at T = 1, where IEEE division returns d
// exactly
SJD_DEV float over_T(float d, float T) { return T == 1.0f ? d : d / T; }
// The same with T = 1 decided at compile time: in a loop, over_T's division
// is computed and then discarded by a select; loops run once per case
// through with_unit_T instead.
template <bool UT>
SJD_DEV float div_T(float d, float T) { return UT ? d : d / T; }
template <class F>
SJD_DEV void with_unit_T(float T, F&& f) {
  if (T == 1.0f) f(std::true_type{});
  else f(std::false_type{});
}

SJD_DEV float comp(const float4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; }
SJD_DEV uint32_t compu(const uint4& v, int e) { return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w; }
SJD_DEV uint64_t pack_key(float key, int x) { return ((uint64_t)__float_as_uint(key) << 32) | (uint32_t)x; }
// order-preserving key with -0 folded onto +0 (logits compare as floats)
SJD_DEV uint32_t okey(float f) { return fkey(f + 0.0f); }

// ---------------------------------------------------------- row statistics
struct RowStats {
  float m;       // largest logit
  float T;
  float tau_v;   // value of the k-th kept logit
  int tau_x;     // its index: kept = l > tau_v or (l == tau_v and x <= tau_x)
  bool all;      // every entry kept
  double invZ;   // 1 / sum of kept weights
  SJD_DEV bool in_set(float l, int x) const { return all || l > tau_v || (l == tau_v && x <= tau_x); }
  SJD_DEV float prob(float l, int x) const {
    if (!in_set(l, x)) return 0.0f;
    const float w = expf(over_T(l - m, T));
    return (float)((double)w * invZ);
  }
};

// The row in registers: chunk c = tid + i * BLOCK holds entries 4c .. 4c+3.
template <int BLOCK, int NC>
SJD_DEV void load_row(float4 (&v)[NC], const float* row, int V) {
  const float4* g = (const float4*)row;
  const int nchunk = V >> 2;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = threadIdx.x + i * BLOCK;
    v[i] = c < nchunk ? g[c] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  }
}

// Radix select (fallback): k-th largest by (value desc, index asc) over
// order-preserving keys (11 + 11 + 10 bits), then over the indices of the
// entries tied at the threshold key (11 + 11 bits).
template <int BLOCK, int NC>
SJD_DEV void radix_topk(const float4 (&v)[NC], int V, int k, VSh<BLOCK, NC>& sh, float& tau_v, int& tau_x) {
  constexpr int W = BLOCK / kWave;
  const int tid = threadIdx.x;
  const int nchunk = V >> 2;
  uint32_t prefix = 0, pmask = 0;
  int rem = k, last_bin = 0;
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const int nb = pass == 2 ? 1024 : 2048;
    for (int b = tid; b < nb; b += BLOCK) sh.o.hist[b] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = tid + i * BLOCK;
      if (c < nchunk) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t key = okey(comp(v[i], e));
          if ((key & pmask) == prefix) atomicAdd(&sh.o.hist[(key >> shift) & (uint32_t)(nb - 1)], 1u);
        }
      }
    }
    __syncthreads();
    const int per = nb / BLOCK > 0 ? nb / BLOCK : 1;
    int s = 0;
    int cnts[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int bi = tid * per + i;
      cnts[i] = (i < per && bi < nb) ? (int)sh.o.hist[nb - 1 - bi] : 0;
      s += cnts[i];
    }
    int run = block_excl_scan<W>(s, sh.red_i);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < per && run < rem && run + cnts[i] >= rem) {
        sh.bin[0] = nb - 1 - (tid * per + i);
        sh.above[0] = run;
      }
      run += cnts[i];
    }
    __syncthreads();
    last_bin = sh.bin[0];
    prefix |= (uint32_t)last_bin << shift;
    pmask |= (uint32_t)(nb - 1) << shift;
    rem -= sh.above[0];
    __syncthreads();
  }
  const int eq = (int)sh.o.hist[last_bin];
  __syncthreads();
  tau_v = 0.0f;
  // value of the threshold key (any entry with that key)
  {
    const uint32_t u = (prefix & 0x80000000u) ? (prefix & 0x7FFFFFFFu) : ~prefix;
    tau_v = __uint_as_float(u);
  }
  if (rem >= eq) {
    tau_x = 0x7FFFFFFF;
    return;
  }
  uint32_t ipre = 0, imask = 0;
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 11 : 0;
    for (int b = tid; b < 2048; b += BLOCK) sh.o.hist[b] = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = tid + i * BLOCK;
      if (c < nchunk) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t x = (uint32_t)(4 * c + e);
          if (okey(comp(v[i], e)) == prefix && (x & imask) == ipre) atomicAdd(&sh.o.hist[(x >> shift) & 2047u], 1u);
        }
      }
    }
    __syncthreads();
    const int per = 2048 / BLOCK;
    int s = 0;
    int cnts[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      cnts[i] = i < per ? (int)sh.o.hist[tid * per + i] : 0;
      s += cnts[i];
    }
    int run = block_excl_scan<W>(s, sh.red_i);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < per && run < rem && run + cnts[i] >= rem) {
        sh.bin[0] = tid * per + i;
        sh.above[0] = run;
      }
      run += cnts[i];
    }
    __syncthreads();
    ipre |= (uint32_t)sh.bin[0] << shift;
    imask |= 2047u << shift;
    rem -= sh.above[0];
    __syncthreads();
  }
  tau_x = (int)ipre;
}

// Block-wide largest value of the row in registers and its smallest value
// above -inf.
template <int BLOCK, int NC>
SJD_DEV void row_maxmin(const float4 (&v)[NC], VSh<BLOCK, NC>& sh, float& mx, float& mn) {
  constexpr int W = BLOCK / kWave;
  mx = -INFINITY;
  mn = INFINITY;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    mx = vmax(mx, vmax(vmax(v[i].x, v[i].y), vmax(v[i].z, v[i].w)));
    mn = vmin(mn, vmin(vmin(v[i].x, v[i].y), vmin(v[i].z, v[i].w)));
  }
  block_maxmin<W>(mx, mn, sh.red_f);
  if (mn == -INFINITY) {
    // rows with -inf entries (padding, masked tokens): minimum over the rest
    mn = INFINITY;
    float t = -INFINITY;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float l = comp(v[i], e);
        if (l > -INFINITY) mn = vmin(mn, l);
      }
    }
    block_maxmin<W>(t, mn, sh.red_f);
  }
}

// Bitmap of a kept set given by the threshold (tau_v, tau_x); the eight
// chunks of a bitmap word belong to eight consecutive lanes, which OR their
// nibbles together.
template <int BLOCK, int NC>
SJD_DEV void bitmap_from_tau(const float4 (&v)[NC], int V, const RowStats& st, uint32_t* bm) {
  const int tid = threadIdx.x;
  const int nchunk = V >> 2;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = tid + i * BLOCK;
    uint32_t bits = 0;
    if (c < nchunk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) bits |= (st.in_set(comp(v[i], e), 4 * c + e) ? 1u : 0u) << e;
    }
    bits <<= 4 * (tid & 7);
    bits = or8_dpp(bits);
    if ((tid & 7) == 0) bm[(tid >> 3) + i * (BLOCK / 8)] = bits;
  }
}

// Exact top-k selection of the row in registers: fills the bitmap bm of the
// kept set and its prefix popcounts pre, sets st.all / tau_v / tau_x (the
// k-th kept entry: kept = l > tau_v or (l == tau_v and x <= tau_x)) and
// returns the number of kept entries.
template <int BLOCK, int NC>
SJD_DEV int select_kept(const float4 (&v)[NC], int V, int top_k, float mx, float mn, VSh<BLOCK, NC>& sh,
                        uint32_t* bm, int32_t* pre, RowStats& st) {
  constexpr int W = BLOCK / kWave;
  constexpr int NW = VSh<BLOCK, NC>::NW;
  const int tid = threadIdx.x;
  const int nchunk = V >> 2;
  const int k = (top_k <= 0 || top_k >= V) ? V : top_k;
  st.all = (k >= V);
  st.tau_v = -INFINITY;
  st.tau_x = 0x7FFFFFFF;
  bool have_bitmap = false;
  if (!st.all) {
    bool fast = (mx < INFINITY) && (mn < INFINITY) && (mx > mn);
    const float scale = fast ? (float)kBins / (mx - mn) : 0.0f;
    fast = fast && (scale < INFINITY) && (scale > 0.0f);
    if (fast) {
      for (int b = tid; b < kBins; b += BLOCK) sh.o.hist[b] = 0;
      for (int b = tid; b < kCandCap + 8; b += BLOCK) {
        sh.o.cand_v[0][b] = -INFINITY;
        sh.o.cand_x[0][b] = 0x7FFFFFFF;
      }
      if (tid == 0) sh.ncand[0] = 0;
      __syncthreads();
      // bin of a value: (l - mn) * scale rounded once (fma), clamped to
      // [0, kBins - 1] (one med3), truncated; monotone in l, so every entry
      // of a higher bin outranks every entry of a lower one (-inf lands in
      // bin 0, +inf in the last)
      const float off = -mn * scale;
      auto binof = [&](float l) -> int {
        return (int)__builtin_amdgcn_fmed3f(__builtin_fmaf(l, scale, off), 0.0f, (float)(kBins - 1));
      };
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int c = tid + i * BLOCK;
        if (c < nchunk) {
#pragma unroll
          for (int e = 0; e < 4; ++e) atomicAdd(&sh.o.hist[binof(comp(v[i], e))], 1u);
        }
      }
      __syncthreads();
      // bins from the top: thread t owns reversed bins [t*per, t*per+per)
      constexpr int per = kBins / BLOCK;
      int cnts[per];
      int s = 0;
#pragma unroll
      for (int i = 0; i < per; ++i) {
        cnts[i] = (int)sh.o.hist[kBins - 1 - (tid * per + i)];
        s += cnts[i];
      }
      int run = block_excl_scan<W>(s, sh.red_i);
#pragma unroll
      for (int i = 0; i < per; ++i) {
        if (run < k && run + cnts[i] >= k) {
          sh.bin[0] = kBins - 1 - (tid * per + i);
          sh.above[0] = run;
        }
        run += cnts[i];
      }
      __syncthreads();
      const int bstar = sh.bin[0], rem = k - sh.above[0], c = (int)sh.o.hist[bstar];
      if (c <= kCandCap) {
        // entries of higher bins are kept; the threshold bin's are collected
#pragma unroll
        for (int i = 0; i < NC; ++i) {
          const int ch = tid + i * BLOCK;
          uint32_t bits = 0, hit = 0;
          if (ch < nchunk) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int b = binof(comp(v[i], e));
              bits |= (b > bstar ? 1u : 0u) << e;
              hit |= (b == bstar ? 1u : 0u) << e;
            }
          }
          if (hit) {  // rare: one branch per chunk, not per entry
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              if ((hit >> e) & 1u) {
                const int p = atomicAdd(&sh.ncand[0], 1);
                sh.o.cand_v[0][p] = comp(v[i], e);
                sh.o.cand_x[0][p] = 4 * ch + e;
              }
            }
          }
          bits <<= 4 * (tid & 7);
          bits = or8_dpp(bits);
          if ((tid & 7) == 0) bm[(tid >> 3) + i * (BLOCK / 8)] = bits;
        }
        __syncthreads();
        // exact rank inside the threshold bin; the first rem join the set
        // (entries past c are sentinels, so the inner loop runs in blocks
        // of eight whose loads issue together)
        const int cpad = (c + 7) & ~7;
        for (int i = tid; i < c; i += BLOCK) {
          const float vi = sh.o.cand_v[0][i];
          const int xi = sh.o.cand_x[0][i];
          int r = 0;
          for (int j0 = 0; j0 < cpad; j0 += 8) {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const float vj = sh.o.cand_v[0][j0 + u];
              r += (vj > vi) || (vj == vi && sh.o.cand_x[0][j0 + u] < xi);
            }
          }
          if (r < rem) atomicOr(&bm[xi >> 5], 1u << (xi & 31));
          if (r == rem - 1) {
            sh.tau_v[0] = vi;
            sh.tau_x[0] = xi;
          }
        }
        __syncthreads();
        st.tau_v = sh.tau_v[0];
        st.tau_x = sh.tau_x[0];
        have_bitmap = true;
      } else {
        fast = false;
      }
    }
    if (!fast) radix_topk<BLOCK, NC>(v, V, k, sh, st.tau_v, st.tau_x);
  }
  if (!have_bitmap) {
    bitmap_from_tau<BLOCK, NC>(v, V, st, bm);
    __syncthreads();
  }
  // per-word prefix popcounts (words contiguous per thread)
  constexpr int WPT = NW / BLOCK > 0 ? NW / BLOCK : 1;
  int cnt[WPT];
  int s = 0;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    cnt[i] = wi < NW ? __popc(bm[wi]) : 0;
    s += cnt[i];
  }
  int run = block_excl_scan<W>(s, sh.red_i);
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    if (wi < NW) pre[wi] = run;
    run += cnt[i];
  }
  if (tid == BLOCK - 1) sh.ncand[0] = run;
  __syncthreads();
  const int total = sh.ncand[0];
  __syncthreads();
  return total;
}

// Kept entries of the row in registers, by rank: ox[r] = index (if ox),
// ol[r] = value.
template <int BLOCK, int NC>
SJD_DEV void compact_row(const float4 (&v)[NC], int V, const uint32_t* bm, const int32_t* pre, uint16_t* ox,
                         float* ol) {
  const int nchunk = V >> 2;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = threadIdx.x + i * BLOCK;
    if (c < nchunk) {
      const uint32_t word = bm[c >> 3];
      const int sh4 = 4 * (c & 7);
      const uint32_t nib = (word >> sh4) & 15u;
      if (nib) {
        int r = pre[c >> 3] + __popc(word & ((1u << sh4) - 1u));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if ((nib >> e) & 1u) {
            if (ox) ox[r] = (uint16_t)(4 * c + e);
            ol[r] = comp(v[i], e);
            ++r;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------ two rows at once
// A spine row whose draft distribution is not cached selects its target row
// (registers v) and its draft row (registers u) together: the same passes
// with one set of barriers and two independent instruction streams. The
// kept sets, ranks, thresholds and normalisers are those the one-row
// functions give (same per-thread orders, same reduction trees).

template <int W>
SJD_DEV void block_maxmin2(float (&mx)[2], float (&mn)[2], float* red) {
  float a0 = wave_max_dpp(mx[0]), a1 = wave_max_dpp(mx[1]);
  float b0 = wave_max_dpp(-mn[0]), b1 = wave_max_dpp(-mn[1]);
  const int w = threadIdx.x / kWave;
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) {
    red[w] = a0;
    red[W + w] = a1;
    red[2 * W + w] = b0;
    red[3 * W + w] = b1;
  }
  __syncthreads();
  a0 = red[0];
  a1 = red[W];
  b0 = red[2 * W];
  b1 = red[3 * W];
#pragma unroll
  for (int i = 1; i < W; ++i) {
    a0 = fmaxf(a0, red[i]);
    a1 = fmaxf(a1, red[W + i]);
    b0 = fmaxf(b0, red[2 * W + i]);
    b1 = fmaxf(b1, red[3 * W + i]);
  }
  mx[0] = a0;
  mx[1] = a1;
  mn[0] = -b0;
  mn[1] = -b1;
  __syncthreads();
}

template <int W>
SJD_DEV void block_excl_scan2(int& a, int& b, int* red) {
  const int ia = wave_incl_scan_dpp(a), ib = wave_incl_scan_dpp(b);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == kWave - 1) {
    red[w] = ia;
    red[W + w] = ib;
  }
  __syncthreads();
  int ba = 0, bb = 0;
  for (int i = 0; i < w; ++i) {
    ba += red[i];
    bb += red[W + i];
  }
  __syncthreads();
  a = ba + ia - a;
  b = bb + ib - b;
}

template <int W>
SJD_DEV void block_sum_d2(double& a, double& b, double* red) {
  a = wave_sum_d_dpp(a);
  b = wave_sum_d_dpp(b);
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    red[w] = a;
    red[W + w] = b;
  }
  __syncthreads();
  double ra = 0.0, rb = 0.0;
#pragma unroll
  for (int i = 0; i < W; ++i) {
    ra += red[i];
    rb += red[W + i];
  }
  __syncthreads();
  a = ra;
  b = rb;
}

// Largest value and smallest value above -inf of both rows.
template <int BLOCK, int NC>
SJD_DEV void row_maxmin2(const float4 (&v)[NC], const float4 (&u)[NC], VSh<BLOCK, NC>& sh, float (&mx)[2],
                         float (&mn)[2]) {
  constexpr int W = BLOCK / kWave;
  mx[0] = mx[1] = -INFINITY;
  mn[0] = mn[1] = INFINITY;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    mx[0] = vmax(mx[0], vmax(vmax(v[i].x, v[i].y), vmax(v[i].z, v[i].w)));
    mn[0] = vmin(mn[0], vmin(vmin(v[i].x, v[i].y), vmin(v[i].z, v[i].w)));
    mx[1] = vmax(mx[1], vmax(vmax(u[i].x, u[i].y), vmax(u[i].z, u[i].w)));
    mn[1] = vmin(mn[1], vmin(vmin(u[i].x, u[i].y), vmin(u[i].z, u[i].w)));
  }
  block_maxmin2<W>(mx, mn, sh.red_f);
  if (mn[0] == -INFINITY || mn[1] == -INFINITY) {
    float t[2] = {-INFINITY, -INFINITY}, m2[2] = {INFINITY, INFINITY};
#pragma unroll
    for (int i = 0; i < NC; ++i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = comp(v[i], e), b = comp(u[i], e);
        if (a > -INFINITY) m2[0] = vmin(m2[0], a);
        if (b > -INFINITY) m2[1] = vmin(m2[1], b);
      }
    }
    block_maxmin2<W>(t, m2, sh.red_f);
    if (mn[0] == -INFINITY) mn[0] = m2[0];
    if (mn[1] == -INFINITY) mn[1] = m2[1];
  }
}

// Top-k selection of both rows by the histogram path. Returns false, with
// nothing decided, when either row needs the one-row path (every entry kept,
// a degenerate value range, or more than kCandCap entries in a threshold
// bin); the decision is uniform over the workgroup.
template <int BLOCK, int NC>
SJD_DEV bool select_kept2(const float4 (&v)[NC], const float4 (&u)[NC], int V, int top_k, const float (&mx)[2],
                          const float (&mn)[2], VSh<BLOCK, NC>& sh, RowStats& ps, RowStats& qs, int& nk,
                          int& nq) {
  constexpr int W = BLOCK / kWave;
  constexpr int NW = VSh<BLOCK, NC>::NW;
  const int tid = threadIdx.x;
  const int nchunk = V >> 2;
  const int k = (top_k <= 0 || top_k >= V) ? V : top_k;
  if (k >= V) return false;
  float scale[2], off[2];
  bool fast = true;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    bool f = (mx[r] < INFINITY) && (mn[r] < INFINITY) && (mx[r] > mn[r]);
    scale[r] = f ? (float)kBins / (mx[r] - mn[r]) : 0.0f;
    f = f && (scale[r] < INFINITY) && (scale[r] > 0.0f);
    fast = fast && f;
    off[r] = -mn[r] * scale[r];
  }
  if (!fast) return false;
  for (int b = tid; b < kBins; b += BLOCK) {
    sh.o.hist[b] = 0;
    sh.o.hist_q[b] = 0;
  }
  for (int b = tid; b < kCandCap + 8; b += BLOCK) {
    sh.o.cand_v[0][b] = -INFINITY;
    sh.o.cand_x[0][b] = 0x7FFFFFFF;
    sh.o.cand_v[1][b] = -INFINITY;
    sh.o.cand_x[1][b] = 0x7FFFFFFF;
  }
  if (tid == 0) {
    sh.ncand[0] = 0;
    sh.ncand[1] = 0;
  }
  __syncthreads();
  auto binof = [&](float l, int r) -> int {
    return (int)__builtin_amdgcn_fmed3f(__builtin_fmaf(l, scale[r], off[r]), 0.0f, (float)(kBins - 1));
  };
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int c = tid + i * BLOCK;
    if (c < nchunk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        atomicAdd(&sh.o.hist[binof(comp(v[i], e), 0)], 1u);
        atomicAdd(&sh.o.hist_q[binof(comp(u[i], e), 1)], 1u);
      }
    }
  }
  __syncthreads();
  constexpr int per = kBins / BLOCK;
  int cp[per], cq[per];
  int sp = 0, sq = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    cp[i] = (int)sh.o.hist[kBins - 1 - (tid * per + i)];
    cq[i] = (int)sh.o.hist_q[kBins - 1 - (tid * per + i)];
    sp += cp[i];
    sq += cq[i];
  }
  block_excl_scan2<W>(sp, sq, sh.red_i);
#pragma unroll
  for (int i = 0; i < per; ++i) {
    if (sp < k && sp + cp[i] >= k) {
      sh.bin[0] = kBins - 1 - (tid * per + i);
      sh.above[0] = sp;
    }
    if (sq < k && sq + cq[i] >= k) {
      sh.bin[1] = kBins - 1 - (tid * per + i);
      sh.above[1] = sq;
    }
    sp += cp[i];
    sq += cq[i];
  }
  __syncthreads();
  const int bs0 = sh.bin[0], bs1 = sh.bin[1];
  const int rem0 = k - sh.above[0], rem1 = k - sh.above[1];
  const int c0 = (int)sh.o.hist[bs0], c1 = (int)sh.o.hist_q[bs1];
  if (c0 > kCandCap || c1 > kCandCap) return false;
  // entries of higher bins are kept; the threshold bins' are collected
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int ch = tid + i * BLOCK;
    uint32_t bp = 0, bq = 0, hp = 0, hq = 0;
    if (ch < nchunk) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int b0 = binof(comp(v[i], e), 0), b1 = binof(comp(u[i], e), 1);
        bp |= (b0 > bs0 ? 1u : 0u) << e;
        hp |= (b0 == bs0 ? 1u : 0u) << e;
        bq |= (b1 > bs1 ? 1u : 0u) << e;
        hq |= (b1 == bs1 ? 1u : 0u) << e;
      }
    }
    if (hp | hq) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if ((hp >> e) & 1u) {
          const int p = atomicAdd(&sh.ncand[0], 1);
          sh.o.cand_v[0][p] = comp(v[i], e);
          sh.o.cand_x[0][p] = 4 * ch + e;
        }
        if ((hq >> e) & 1u) {
          const int p = atomicAdd(&sh.ncand[1], 1);
          sh.o.cand_v[1][p] = comp(u[i], e);
          sh.o.cand_x[1][p] = 4 * ch + e;
        }
      }
    }
    bp <<= 4 * (tid & 7);
    bq <<= 4 * (tid & 7);
    bp = or8_dpp(bp);
    bq = or8_dpp(bq);
    if ((tid & 7) == 0) {
      sh.bm[(tid >> 3) + i * (BLOCK / 8)] = bp;
      sh.o.bmq[(tid >> 3) + i * (BLOCK / 8)] = bq;
    }
  }
  __syncthreads();
  // exact rank inside each threshold bin; the first rem join the set
  for (int t = tid; t < c0 + c1; t += BLOCK) {
    const int r = t < c0 ? 0 : 1;
    const int i = t - (r ? c0 : 0);
    const int c = r ? c1 : c0;
    const float vi = sh.o.cand_v[r][i];
    const int xi = sh.o.cand_x[r][i];
    int rank = 0;
    for (int j0 = 0; j0 < c; j0 += 8) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float vj = sh.o.cand_v[r][j0 + q];
        rank += (vj > vi) || (vj == vi && sh.o.cand_x[r][j0 + q] < xi);
      }
    }
    const int rem = r ? rem1 : rem0;
    if (rank < rem) atomicOr(r ? &sh.o.bmq[xi >> 5] : &sh.bm[xi >> 5], 1u << (xi & 31));
    if (rank == rem - 1) {
      sh.tau_v[r] = vi;
      sh.tau_x[r] = xi;
    }
  }
  __syncthreads();
  ps.all = qs.all = false;
  ps.tau_v = sh.tau_v[0];
  ps.tau_x = sh.tau_x[0];
  qs.tau_v = sh.tau_v[1];
  qs.tau_x = sh.tau_x[1];
  // per-word prefix popcounts of both bitmaps
  constexpr int WPT = NW / BLOCK > 0 ? NW / BLOCK : 1;
  int np[WPT], nqw[WPT];
  int rp = 0, rq = 0;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    np[i] = wi < NW ? __popc(sh.bm[wi]) : 0;
    nqw[i] = wi < NW ? __popc(sh.o.bmq[wi]) : 0;
    rp += np[i];
    rq += nqw[i];
  }
  block_excl_scan2<W>(rp, rq, sh.red_i);
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    if (wi < NW) {
      sh.pre[wi] = rp;
      sh.o.preq[wi] = rq;
    }
    rp += np[i];
    rq += nqw[i];
  }
  if (tid == BLOCK - 1) {
    sh.ncand[0] = rp;
    sh.ncand[1] = rq;
  }
  __syncthreads();
  nk = sh.ncand[0];
  nq = sh.ncand[1];
  __syncthreads();
  return true;
}

// ------------------------------------------------------ candidate path
// Top-k selection that touches each logit once. A sample of the row (every
// fourth entry of half the register slots) gives a value lo that about
// k + 3 sigma of the row's entries reach; one pass over the row in registers
// appends every entry >= lo to its wave's region of LDS (per-wave append by
// ballot and mbcnt). The exact threshold (value desc, index asc) is then
// found among those candidates alone: a histogram over [lo, max], the
// threshold bin's entries ranked exactly. The kept set, its normaliser and
// the threshold are those of the full selection; only the order of the fp64
// normaliser sum differs. The compact list (index order) is built from the
// candidates when a row draws from it (fast_build_list). Any case the
// candidates cannot decide (a row with -inf, NaN or +inf entries, too few or
// too many candidates, a crowded threshold bin, tied draft values split by
// the threshold) returns false with nothing decided; the caller then runs
// the full selection.

// Wave max that propagates NaN (no quieting copy per step).
SJD_DEV float wave_vmax_dpp(float v) {
  return wave_reduce32(v, [](float a, float b) { return __builtin_elementwise_maximum(a, b); });
}

// Block-wide max of four values; every thread gets the four results.
template <int W>
SJD_DEV void block_max4(float (&a)[4], float* red) {
  const int w = threadIdx.x / kWave;
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = wave_vmax_dpp(a[i]);
  if ((threadIdx.x & (kWave - 1)) == 0) *(float4*)&red[4 * w] = make_float4(a[0], a[1], a[2], a[3]);
  __syncthreads();
  float4 m = *(const float4*)&red[0];
#pragma unroll 2
  for (int t = 1; t < W; ++t) {
    const float4 o = *(const float4*)&red[4 * t];
    m.x = __builtin_elementwise_maximum(m.x, o.x);
    m.y = __builtin_elementwise_maximum(m.y, o.y);
    m.z = __builtin_elementwise_maximum(m.z, o.z);
    m.w = __builtin_elementwise_maximum(m.w, o.w);
  }
  a[0] = m.x; a[1] = m.y; a[2] = m.z; a[3] = m.w;
  __syncthreads();
}

// One wave: the bin of hist[0..NB) (counted from the top) that holds the
// target-th entry, and the number of entries above it, into *bin / *above.
template <int NB>
SJD_DEV void wave_find_from_top(const uint32_t* hist, int target, int* bin, int* above) {
  constexpr int PER = NB / kWave;
  static_assert(PER % 4 == 0, "bins are read four at a time");
  const int lane = threadIdx.x & (kWave - 1);
  // lane l owns bins [NB - (l + 1) * PER, NB - l * PER), read from the top
  uint32_t c[PER];
#pragma unroll
  for (int i = 0; i < PER; i += 4) {
    const uint4 q = *(const uint4*)&hist[NB - (lane + 1) * PER + i];
    c[PER - 1 - i] = q.x; c[PER - 2 - i] = q.y; c[PER - 3 - i] = q.z; c[PER - 4 - i] = q.w;
  }
  int s = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) s += (int)c[i];
  int run = wave_incl_scan_dpp(s) - s;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (run < target && run + (int)c[i] >= target) {
      *bin = NB - 1 - (lane * PER + i);
      *above = run;
    }
    run += (int)c[i];
  }
}

template <int BLOCK, int NC, bool TWO>
SJD_DEV bool fast_select(const float4 (&v)[NC], const float4 (&u)[NC], int V, int top_k, float T,
                         VSh<BLOCK, NC>& sh, RowStats& ps, RowStats& qs, float lp0, float lq0, float& ep0,
                         float& eq0) {
  using Sh = VSh<BLOCK, NC>;
  constexpr int W = BLOCK / kWave;
  constexpr int CAPW = Sh::CAPW;
  constexpr int R = TWO ? 2 : 1;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int nchunk = V >> 2;
  const int k = (top_k <= 0 || top_k >= V) ? V : top_k;
  if (k >= V) return false;

  // 1. row maxima, and the smallest sampled value (entry 4c of the even
  //    slots); the samples are binned over [sample min, row max]
  float st[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    st[0] = vmax(st[0], vmax(vmax(v[i].x, v[i].y), vmax(v[i].z, v[i].w)));
    if (TWO) st[2] = vmax(st[2], vmax(vmax(u[i].x, u[i].y), vmax(u[i].z, u[i].w)));
    if ((i & 1) == 0 && tid + i * BLOCK < nchunk) {
      st[1] = vmax(st[1], -v[i].x);
      if (TWO) st[3] = vmax(st[3], -u[i].x);
    }
  }
  block_max4<W>(st, sh.red_f);
  // the first candidate's weights under both rows' maxima, computed here so
  // that the accept test after the selection only scales them
  ep0 = expf(over_T(lp0 - st[0], T));
  if (TWO) eq0 = expf(over_T(lq0 - st[2], T));
  // samples per row
  int S = 0;
#pragma unroll
  for (int i = 0; i < NC; i += 2) {
    const int n = nchunk - i * BLOCK;
    S += n <= 0 ? 0 : (n >= BLOCK ? BLOCK : n);
  }
  // rank (from the top) of the sample that sets lo: k's share of the
  // samples plus three standard deviations (scales and ranks here only steer
  // the selection, so approximate reciprocals do)
  const float kf = (float)k, rV = __builtin_amdgcn_rcpf((float)V);
  const float kSV = kf * (float)S * rV;
  const int rstar = (int)ceilf(kSV + 3.0f * __builtin_amdgcn_sqrtf(kSV * (1.0f - kf * rV)) + 1.0f);
  if (rstar > S) return false;
  float sscale[2], soff[2], smn[2], srng[2];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const float mx = st[2 * r];
    smn[r] = -st[2 * r + 1];
    // finite range (a -inf, +inf or NaN sample or maximum sends the row to
    // the full selection)
    if (!(mx > smn[r]) || !(mx < INFINITY) || !(smn[r] > -INFINITY)) return false;
    srng[r] = mx - smn[r];
    sscale[r] = (float)kSampBins * __builtin_amdgcn_rcpf(srng[r]);
    if (!(sscale[r] < INFINITY) || !(sscale[r] > 0.0f)) return false;
    soff[r] = -smn[r] * sscale[r];
  }

  // 2. sample histograms; lo = one bin below the bin that holds sample rstar
  //    from the top
  for (int b = tid; b < R * kFastBins; b += BLOCK) (&sh.f.hist[0][0])[b] = 0;
  __syncthreads();
  auto sbin = [&](float l, int r) -> int {
    return (int)__builtin_amdgcn_fmed3f(__builtin_fmaf(l, sscale[r], soff[r]), 0.0f, (float)(kSampBins - 1));
  };
#pragma unroll
  for (int i = 0; i < NC; i += 2) {
    if (tid + i * BLOCK < nchunk) {
      atomicAdd(&sh.f.hist[0][sbin(v[i].x, 0)], 1u);
      if (TWO) atomicAdd(&sh.f.hist[1][sbin(u[i].x, 1)], 1u);
    }
  }
  __syncthreads();
  if (w < R) wave_find_from_top<kSampBins>(sh.f.hist[w], rstar, &sh.bin[w], &sh.above[w]);
  __syncthreads();
  float lo[2];
#pragma unroll
  for (int r = 0; r < R; ++r) lo[r] = smn[r] + ((float)sh.bin[r] - 1.0f) * srng[r] * (1.0f / kSampBins);

  // 3. candidates: every entry >= lo, appended to the wave's region
  //    [w * CAPW, w * CAPW + count); a region that would overflow stops
  //    taking entries and marks the row
  int cnt[2] = {0, 0};
  bool ovf[2] = {false, false};
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    const int xb = 4 * (tid + i * BLOCK);  // padding chunks hold -inf and are never taken
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float4 x4 = r == 0 ? v[i] : u[i];
      const bool s0 = x4.x >= lo[r], s1 = x4.y >= lo[r], s2 = x4.z >= lo[r], s3 = x4.w >= lo[r];
      const uint64_t m0 = __ballot(s0), m1 = __ballot(s1), m2 = __ballot(s2), m3 = __ballot(s3);
      const int t0 = __popcll(m0), t1 = __popcll(m1), t2 = __popcll(m2), t3 = __popcll(m3);
      const int tot = t0 + t1 + t2 + t3;
      if (cnt[r] + tot <= CAPW) {
        int base = w * CAPW + cnt[r];
        auto put = [&](bool s, uint64_t m, float l, int e) {
          if (s) {
            const int p = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)m, (uint32_t)base));
            if (r == 0) {
              sh.f.cv[p] = l;
              sh.f.cx[p] = xb + e;
              if (TWO) sh.f.cq[p] = comp(u[i], e);
            } else {
              sh.u.dv[p] = l;
            }
          }
        };
        put(s0, m0, x4.x, 0);
        base += t0;
        put(s1, m1, x4.y, 1);
        base += t1;
        put(s2, m2, x4.z, 2);
        base += t2;
        put(s3, m3, x4.w, 3);
      } else {
        ovf[r] = true;
      }
      cnt[r] += tot;
    }
  }
  if (lane == 0) {
    sh.wcnt[0][w] = ovf[0] ? -1 : cnt[0];
    if (TWO) sh.wcnt[1][w] = ovf[1] ? -1 : cnt[1];
  }
  __syncthreads();
  int tot[2] = {0, 0};
  bool bad = false;
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int t = 0; t < W; ++t) {
      const int c = sh.wcnt[r][t];
      bad |= c < 0;
      tot[r] += c;
    }
    bad |= tot[r] < k;
  }
  if (bad) {
    __syncthreads();
    return false;
  }

  // 4. histogram of the candidates over [lo, max]
  float scale[2], off[2];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const float mx = st[2 * r];
    scale[r] = (float)kFastBins * __builtin_amdgcn_rcpf(mx - lo[r]);
    if (!(scale[r] < INFINITY) || !(scale[r] > 0.0f)) bad = true;
    off[r] = -lo[r] * scale[r];
  }
  if (bad) {
    __syncthreads();
    return false;
  }
  auto fbin = [&](float l, int r) -> int {
    return (int)__builtin_amdgcn_fmed3f(__builtin_fmaf(l, scale[r], off[r]), 0.0f, (float)(kFastBins - 1));
  };
  for (int b = tid; b < R * kFastBins; b += BLOCK) (&sh.f.hist[0][0])[b] = 0;
  for (int b = tid; b < R * (kCandCap + 8); b += BLOCK) {
    (&sh.f.tb_v[0][0])[b] = -INFINITY;
    (&sh.f.tb_x[0][0])[b] = 0x7FFFFFFF;
  }
  if (tid == 0) {
    sh.ncand[0] = 0;
    sh.ncand[1] = 0;
    sh.fflag = 0;
  }
  __syncthreads();
  for (int i = lane; i < cnt[0]; i += kWave) atomicAdd(&sh.f.hist[0][fbin(sh.f.cv[w * CAPW + i], 0)], 1u);
  if (TWO)
    for (int i = lane; i < cnt[1]; i += kWave) atomicAdd(&sh.f.hist[1][fbin(sh.u.dv[w * CAPW + i], 1)], 1u);
  __syncthreads();
  if (w < R) wave_find_from_top<kFastBins>(sh.f.hist[w], k, &sh.bin[w], &sh.above[w]);
  __syncthreads();
  int bs[2], rem[2], cb[2];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    bs[r] = sh.bin[r];
    rem[r] = k - sh.above[r];
    cb[r] = (int)sh.f.hist[r][bs[r]];
    bad |= cb[r] > kCandCap;
  }
  if (bad) {
    __syncthreads();
    return false;
  }

  // 5. one pass over the candidates: entries of bins above the threshold bin
  //    are kept (weight into the normaliser; a target candidate's slot keeps
  //    its weight), entries below it are not (slot -1), the threshold bin's
  //    entries are collected with their slot
  const float mp = st[0], mq = st[2];
  double zp = 0.0, zq = 0.0;
  with_unit_T(T, [&](auto ut) {
    constexpr bool UT = decltype(ut)::value;
    for (int i = lane; i < cnt[0]; i += kWave) {
      const int s = w * CAPW + i;
      const float l = sh.f.cv[s];
      const int bn = fbin(l, 0);
      float e = -1.0f;
      if (bn > bs[0]) {
        e = expf(div_T<UT>(l - mp, T));
        zp += (double)e;
      } else if (bn == bs[0]) {
        const int p = atomicAdd(&sh.ncand[0], 1);
        sh.f.tb_v[0][p] = l;
        sh.f.tb_x[0][p] = sh.f.cx[s];
        sh.f.tb_s[0][p] = s;
      }
      sh.f.cv[s] = e;
    }
    if (TWO) {
      for (int i = lane; i < cnt[1]; i += kWave) {
        const int s = w * CAPW + i;
        const float l = sh.u.dv[s];
        const int bn = fbin(l, 1);
        if (bn > bs[1]) {
          zq += (double)expf(div_T<UT>(l - mq, T));
        } else if (bn == bs[1]) {
          const int p = atomicAdd(&sh.ncand[1], 1);
          sh.f.tb_v[1][p] = l;
          sh.f.tb_x[1][p] = s;
        }
      }
    }
  });
  __syncthreads();
  // 6. exact rank inside each threshold bin: the first rem join the kept set
  //    (and the normaliser), entry rem - 1 is the threshold
  const int c0 = cb[0], c1 = TWO ? cb[1] : 0;
  for (int t = tid; t < c0 + c1; t += BLOCK) {
    const int r = t < c0 ? 0 : 1;
    const int i = t - (r ? c0 : 0);
    const int c = r ? c1 : c0;
    const float vi = sh.f.tb_v[r][i];
    const int xi = sh.f.tb_x[r][i];
    int rank = 0, later_tie = 0;
    for (int j0 = 0; j0 < c; j0 += 8) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float vj = sh.f.tb_v[r][j0 + q];
        const int xj = sh.f.tb_x[r][j0 + q];
        rank += (vj > vi) || (vj == vi && xj < xi);
        later_tie += (vj == vi && xj > xi);
      }
    }
    const bool keep = rank < rem[r];
    const float e = keep ? expf(over_T(vi - (r ? mq : mp), T)) : -1.0f;
    if (r == 0) {
      sh.f.cv[sh.f.tb_s[0][i]] = e;
      if (keep) zp += (double)e;
    } else if (keep) {
      zq += (double)e;
    }
    if (rank == rem[r] - 1) {
      sh.tau_v[r] = vi;
      sh.tau_x[r] = r == 0 ? xi : 0x7FFFFFFF;
      // a draft value tied across the threshold needs token indices
      if (r == 1 && later_tie > 0) sh.fflag = 1;
    }
  }
  block_sum_d2<W>(zp, zq, sh.red_d);  // (its barriers publish tau and fflag)
  if (sh.fflag) {
    __syncthreads();
    return false;
  }
  ps.m = mp;
  ps.T = T;
  ps.all = false;
  ps.tau_v = sh.tau_v[0];
  ps.tau_x = sh.tau_x[0];
  ps.invZ = 1.0 / zp;
  if (TWO) {
    qs.m = mq;
    qs.T = T;
    qs.all = false;
    qs.tau_v = sh.tau_v[1];
    qs.tau_x = sh.tau_x[1];
    qs.invZ = 1.0 / zq;
  }
  return true;
}

// Compact list (index order) of the kept target candidates: bitmap of the
// kept set, per-word prefix popcounts, then each kept token at its rank with
// its probability and, if want_q, its draft probability (from the draft
// logits stored beside it, or read from draft_row).
template <int BLOCK, int NC>
SJD_DEV void fast_build_list(VSh<BLOCK, NC>& sh, const RowStats& ps, const RowStats& qs, bool want_q, bool two,
                             const float* draft_row) {
  using Sh = VSh<BLOCK, NC>;
  constexpr int W = BLOCK / kWave;
  constexpr int NW = Sh::NW;
  constexpr int CAPW = Sh::CAPW;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int cnt = sh.wcnt[0][w];
  for (int i = tid; i < NW; i += BLOCK) sh.bm[i] = 0;
  __syncthreads();
  for (int i = lane; i < cnt; i += kWave) {
    const int s = w * CAPW + i;
    if (sh.f.cv[s] >= 0.0f) {
      const int x = sh.f.cx[s];
      atomicOr(&sh.bm[x >> 5], 1u << (x & 31));
    }
  }
  __syncthreads();
  constexpr int WPT = NW / BLOCK > 0 ? NW / BLOCK : 1;
  int wc[WPT];
  int s0 = 0;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    wc[i] = wi < NW ? __popc(sh.bm[wi]) : 0;
    s0 += wc[i];
  }
  int run = block_excl_scan<W>(s0, sh.red_i);
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    if (wi < NW) sh.pre[wi] = run;
    run += wc[i];
  }
  __syncthreads();
  with_unit_T(qs.T, [&](auto ut) {
    constexpr bool UT = decltype(ut)::value;
    for (int i = lane; i < cnt; i += kWave) {
      const int s = w * CAPW + i;
      const float e = sh.f.cv[s];
      if (e >= 0.0f) {
        const int x = sh.f.cx[s];
        const int r = sh.pre[x >> 5] + __popc(sh.bm[x >> 5] & ((1u << (x & 31)) - 1u));
        sh.u.sp.x[r] = (uint16_t)x;
        sh.u.sp.p[r] = (float)((double)e * ps.invZ);
        if (want_q) {
          const float l = two ? sh.f.cq[s] : draft_row[x];
          sh.u.sp.q[r] = qs.in_set(l, x) ? (float)((double)expf(div_T<UT>(l - qs.m, qs.T)) * qs.invZ) : 0.0f;
        }
      }
    }
  });
  __syncthreads();
}

// Softmax weights over a compact list of logits: w[i] = expf((w[i] - m) / T)
// in place; returns 1 / sum (fp64, fixed order).
template <int BLOCK, int NC>
SJD_DEV double softmax_weights(float* w, int n, float m, float T, VSh<BLOCK, NC>& sh) {
  constexpr int W = BLOCK / kWave;
  double z = 0.0;
  for (int i = threadIdx.x; i < n; i += BLOCK) {
    const float e = expf(over_T(w[i] - m, T));
    w[i] = e;
    z += (double)e;
  }
  return 1.0 / block_sum_d<W>(z, sh.red_d);
}

template <int BLOCK, int NC>
SJD_DEV bool kept(const VSh<BLOCK, NC>& sh, int x) { return (sh.bm[x >> 5] >> (x & 31)) & 1u; }
template <int BLOCK, int NC>
SJD_DEV int rank_of(const VSh<BLOCK, NC>& sh, int x) {
  return sh.pre[x >> 5] + __popc(sh.bm[x >> 5] & ((1u << (x & 31)) - 1u));
}

struct Stages {
  int n;        // stages whose residual has been formed
  int cand[8];
  float Nf[8];  // normaliser of p^(s)
  float den[8]; // 1 - q mass of candidates rejected before stage s
  // rho^(n+1)(y): the unnormalised residual after n rejected stages; loops
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

// Race over the compact list: argmin over kept entries with weight w(e) > 0
// of Exp(1) / w, the exponential of entry e being stream element e.
template <int BLOCK, int NC, class Wfn>
SJD_DEV int race_compact(const VSh<BLOCK, NC>& shc, VSh<BLOCK, NC>& sh, int nk, const Stream& rs, Wfn wfn) {
  constexpr int W = BLOCK / kWave;
  uint64_t best = kNoKey;
  for (int j = threadIdx.x; 4 * j < nk; j += BLOCK) {
    const uint4 wd = rs.block((uint32_t)j);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int ent = 4 * j + e;
      if (ent < nk) {
        const float w = wfn(ent);
        if (w > 0.0f) {
          const uint64_t pk = pack_key(exp1(compu(wd, e)) / w, (int)shc.u.sp.x[ent]);
          best = pk < best ? pk : best;
        }
      }
    }
  }
  best = block_min_u64<W>(best, sh.red_u);
  return best == kNoKey ? -1 : (int)(uint32_t)best;
}

// Drafting candidates of one row (proactive drafting, Sec. 4.1): the Km1
// smallest race keys of p over the kept list (sp_x / sp_p, nk entries)
// without token excl, in ascending key order (K - 1 draws without
// replacement), from stream (tag 5, stage 0, row j); out[t] = -1 past the
// tokens found.
template <int BLOCK, int NC, class Sh>
SJD_DEV void draft_candidates(const VerifyArgs& a, Sh& sh, int nk, int excl, int j, int b, int Km1,
                              int (&out)[7]) {
  constexpr int W = BLOCK / kWave;
  const int tid = threadIdx.x;
  const Stream rs(a.seed, kTagPd, 0, (uint32_t)j, (uint32_t)b, a.step);
  // this thread's keys: Philox blocks tid, tid + BLOCK, ... of the compact
  // list (keys carry the token, so they are distinct)
  constexpr int KB = (kKcap / 4 + BLOCK - 1) / BLOCK;
  uint64_t key[4 * KB];
#pragma unroll
  for (int q = 0; q < KB; ++q) {
    const int jj = tid + q * BLOCK;
#pragma unroll
    for (int e = 0; e < 4; ++e) key[4 * q + e] = kNoKey;
    if (4 * jj < nk) {
      const uint4 wd = rs.block((uint32_t)jj);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ent = 4 * jj + e;
        if (ent < nk) {
          const int x = (int)sh.u.sp.x[ent];
          const float pw = sh.u.sp.p[ent];
          if (pw > 0.0f && x != excl) key[4 * q + e] = pack_key(exp1(compu(wd, e)) / pw, x);
        }
      }
    }
  }
  // each wave's Km1 smallest keys in order, then the Km1 smallest of
  // those W lists
  const int lane = tid & (kWave - 1), w = tid / kWave;
  uint64_t mine = kNoKey;
#pragma unroll
  for (int t = 0; t < 7; ++t) {
    if (t < Km1) {
      uint64_t lm = key[0];
#pragma unroll
      for (int q = 1; q < 4 * KB; ++q) lm = key[q] < lm ? key[q] : lm;
      const uint64_t m = wave_min_u64_dpp(lm);
      if (m != kNoKey) {
#pragma unroll
        for (int q = 0; q < 4 * KB; ++q) key[q] = key[q] == m ? kNoKey : key[q];
      }
      if (lane == t) mine = m;
    }
  }
  if (lane < 8) sh.pd_w[w * 8 + lane] = mine;
  __syncthreads();
  if (w == 0) {
    uint64_t c0 = kNoKey, c1 = kNoKey;
    if (lane < W * 8) c0 = sh.pd_w[lane];
    if (lane + kWave < W * 8) c1 = sh.pd_w[lane + kWave];
#pragma unroll
    for (int t = 0; t < 7; ++t) {
      if (t < Km1) {
        const uint64_t m = wave_min_u64_dpp(c0 < c1 ? c0 : c1);
        if (m != kNoKey) {
          if (c0 == m) c0 = kNoKey;
          if (c1 == m) c1 = kNoKey;
        }
        if (lane == 0) sh.pd_o[t] = m == kNoKey ? -1 : (int)(uint32_t)m;
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < 7; ++t) out[t] = t < Km1 ? sh.pd_o[t] : -1;
}

// A row's target statistics in its record (words 10..15), for the rows
// k_verify_pd drafts at.
SJD_DEV void put_stats(int32_t* rec, const RowStats& st) {
  rec[10] = __float_as_int(st.tau_v);
  rec[11] = st.tau_x;
  rec[12] = __float_as_int(st.m);
  const uint64_t z = (uint64_t)__double_as_longlong(st.invZ);
  rec[13] = (int32_t)(uint32_t)z;
  rec[14] = (int32_t)(uint32_t)(z >> 32);
  rec[15] = st.all ? 1 : 0;
}
SJD_DEV RowStats get_stats(const int32_t* rec, float T) {
  RowStats st{};
  st.tau_v = __int_as_float(rec[10]);
  st.tau_x = rec[11];
  st.m = __int_as_float(rec[12]);
  st.invZ = __longlong_as_double((long long)(((uint64_t)(uint32_t)rec[14] << 32) | (uint32_t)rec[13]));
  st.all = rec[15] != 0;
  st.T = T;
  return st;
}

// ------------------------------------------------------------ row kernel
// What a row needs from memory (uniform over the workgroup).
struct RowLoad {
  bool valid;   // the trial's window description is well formed
  bool need_p;  // the row's own logits are used
  bool need_q;  // its draft row is read (a spine row with a valid draft token)
  const float* cur;
  const float* draft;
  const RowStatsCache* q_cached;  // the draft row's statistics from the previous step, or NULL
};

// the logits row of (trial, window row)
SJD_DEV const float* row_logits(const VerifyArgs& a, int row) {
  const int b = row / a.L, j = row % a.L;
  return a.cur + (size_t)b * (a.cur_bstride ? (size_t)a.cur_bstride : (size_t)a.L * a.V) + (size_t)j * a.V;
}

SJD_DEV bool forced_pos(const VerifyArgs& a, long g) {
  return a.row_len > 0 && g >= 0 && (g % (a.row_len + 1)) == a.row_len;
}

SJD_DEV RowLoad plan_load(const VerifyArgs& a, int row) {
  RowLoad r;
  const int b = row / a.L, j = row % a.L;
  const int Km1 = a.K - 1;
  // every word the plan may need that lies in bounds whatever the window
  // says, loaded before any of them is used
  const int32_t* meta = a.in_meta + (size_t)b * trial_stride(a, 4);
  const int D_in = meta[0], n_q = meta[1];
  const long g0 = meta[2];
  const int dtok = a.draft_tok[(size_t)b * trial_stride(a, a.L) + j];
  const int qoff = a.q_off ? a.q_off[(size_t)b * trial_stride(a, 1)] : 0;
  const int n_s = a.L - Km1 * D_in;
  r.valid = !(D_in < 0 || D_in > a.D || a.K * D_in > a.L || n_q < 0 || n_q > n_s);
  r.need_p = false;
  r.need_q = false;
  r.cur = row_logits(a, row);
  r.draft = nullptr;
  r.q_cached = nullptr;
  if (!r.valid) return r;
  if (j < n_s) {
    const bool is_forced = forced_pos(a, g0 + j);
    r.need_p = !is_forced;
    if (!is_forced && j < n_q) {
      const int x0 = dtok - a.vis_lo;
      if (x0 >= 0 && x0 < a.V) {
        r.need_q = true;
        const int qrow = qoff + j;
        r.draft = a.draft + (size_t)b * a.draft_bstride + (size_t)qrow * a.V;
        if (a.stats_in) {
          const RowStatsCache* c = a.stats_in + (size_t)b * a.L + qrow;
          if (c->tag == a.stats_tag - 1u && c->T == a.T && c->top_k == a.top_k) r.q_cached = c;
        }
      }
    }
  } else {
    const int sib_d = (j - n_s) / Km1, sib_k = (j - n_s) % Km1 + 2;
    const int sib_tok = a.sib ? a.sib[(size_t)b * trial_stride(a, (size_t)a.D * Km1) + (size_t)sib_d * Km1 + (sib_k - 2)] : -1;
    r.need_p = !(sib_tok < 0 || forced_pos(a, g0 + sib_d) || forced_pos(a, g0 + sib_d + 1));
  }
  if (a.dbg_p) r.need_p = true;
  return r;
}

// One row. With PF, v already holds the row's logits (if ld.need_p) and vq
// its draft row (if ld.need_q), both loaded at kernel start so that the two
// reads overlap; without PF, vq is v and each row is loaded when needed.
template <int BLOCK, int NC, bool PF>
SJD_DEV void verify_row(const VerifyArgs& a, VSh<BLOCK, NC>& sh, int row, const RowLoad& ld, float4 (&v)[NC],
                        float4 (&vq)[NC]) {
  constexpr int W = BLOCK / kWave;
  const int tid = threadIdx.x;
  const int b = row / a.L, j = row % a.L;
  const int L = a.L, V = a.V, Km1 = a.K - 1;
  const int nchunk = V >> 2;
  if (!ld.valid) return;  // finalize flags the trial
  const int32_t* meta = a.in_meta + (size_t)b * trial_stride(a, 4);
  const int D_in = meta[0];
  const long g0 = meta[2];
  const int n_s = L - Km1 * D_in;
  int32_t* rec = a.rec + ((size_t)b * L + j) * kRecInts;
  const bool ac = (a.flags & kFlagAC) != 0;
  const bool pd = (a.flags & kFlagPD) != 0 && Km1 > 0;
  const bool spine = j < n_s;

  // candidates: the spine draft, then (tree rows) its siblings; an
  // out-of-range or repeated candidate ends the list
  Stages stg;
  stg.n = 0;
#pragma unroll
  for (int t = 0; t < 8; ++t) { stg.cand[t] = -1; stg.Nf[t] = 1.0f; stg.den[t] = 1.0f; }
  int ncand = 0;
  if (spine && ld.need_q) {
    stg.cand[0] = a.draft_tok[(size_t)b * trial_stride(a, L) + j] - a.vis_lo;
    ncand = 1;
    if (j < D_in && a.sib) {
      bool open = true;
#pragma unroll
      for (int k = 0; k < 7; ++k) {
        if (open && k < Km1) {
          int y = a.sib[(size_t)b * trial_stride(a, (size_t)a.D * Km1) + (size_t)j * Km1 + k];
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

  // the draft and target logits at the first candidate, loaded now so that
  // the first accept test does not wait for them (later candidates are read
  // when their stage comes)
  const float qcl0 = ncand > 0 ? ld.draft[stg.cand[0]] : 0.0f;
  const float pcl0 = ncand > 0 ? ld.cur[stg.cand[0]] : 0.0f;
  // the first accept draw (uniform over the workgroup), ahead of the selection
  const float u0 = u01(Stream(a.seed, kTagAcc, 0u, (uint32_t)j, (uint32_t)b, a.step).word(0));
  // candidate path: the first candidate's weights exp((l - max) / T) under
  // each row's maximum (computed once the maxima are known)
  float ep0 = 0.0f, eq0 = 0.0f;

  RowStats ps{}, qs{};
  int nk = 0;
  bool q_ready = false;  // the draft distribution at the target's kept entries is in sp_q
  // candidate path: the compact list (and sp_q) is built when a draw needs it
  bool lazy = false;
  bool fast_first = false;  // ep0 / eq0 hold the first candidate's weights
  const bool two = ld.need_q && !ld.q_cached;
  if (ld.need_p) {
    if (!PF) load_row<BLOCK, NC>(v, ld.cur, V);
    if constexpr (PF) {
      if (!(a.flags & kFlagFullSelect)) {
        if (two) lazy = fast_select<BLOCK, NC, true>(v, vq, V, a.top_k, a.T, sh, ps, qs, pcl0, qcl0, ep0, eq0);
        else lazy = fast_select<BLOCK, NC, false>(v, v, V, a.top_k, a.T, sh, ps, qs, pcl0, qcl0, ep0, eq0);
      }
      if (lazy) {
        nk = (a.top_k <= 0 || a.top_k >= V) ? V : a.top_k;
        q_ready = two;
        fast_first = true;
      } else if (two) {
        // target and draft rows together
        float mx2[2], mn2[2];
        row_maxmin2<BLOCK, NC>(v, vq, sh, mx2, mn2);
        ps.m = mx2[0];
        qs.m = mx2[1];
        ps.T = qs.T = a.T;
        int nq = 0;
        if (select_kept2<BLOCK, NC>(v, vq, V, a.top_k, mx2, mn2, sh, ps, qs, nk, nq)) {
          // target compaction; the draft logits at the target's kept entries
          // (by target rank) and at its own (by draft rank, its normaliser)
#pragma unroll
          for (int i = 0; i < NC; ++i) {
            const int c = tid + i * BLOCK;
            if (c < nchunk) {
              const int sh4 = 4 * (c & 7);
              const uint32_t wp = sh.bm[c >> 3], wq = sh.o.bmq[c >> 3];
              const uint32_t np = (wp >> sh4) & 15u, nqb = (wq >> sh4) & 15u;
              if (np | nqb) {
                int rp = sh.pre[c >> 3] + __popc(wp & ((1u << sh4) - 1u));
                int rq = sh.o.preq[c >> 3] + __popc(wq & ((1u << sh4) - 1u));
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  if ((np >> e) & 1u) {
                    sh.u.sp.x[rp] = (uint16_t)(4 * c + e);
                    sh.u.sp.p[rp] = comp(v[i], e);
                    sh.u.sp.q[rp] = comp(vq[i], e);
                    ++rp;
                  }
                  if ((nqb >> e) & 1u) sh.o.qc[rq++] = comp(vq[i], e);
                }
              }
            }
          }
          __syncthreads();
          double zp = 0.0, zq = 0.0;
          const int nmax = nk > nq ? nk : nq;
          for (int i = tid; i < nmax; i += BLOCK) {
            if (i < nk) {
              const float e = expf(over_T(sh.u.sp.p[i] - ps.m, a.T));
              sh.u.sp.p[i] = e;
              zp += (double)e;
            }
            if (i < nq) zq += (double)expf(over_T(sh.o.qc[i] - qs.m, a.T));
          }
          block_sum_d2<W>(zp, zq, sh.red_d);
          ps.invZ = 1.0 / zp;
          qs.invZ = 1.0 / zq;
          for (int i = tid; i < nk; i += BLOCK) {
            sh.u.sp.p[i] = (float)((double)sh.u.sp.p[i] * ps.invZ);
            const int x = (int)sh.u.sp.x[i];
            const bool in_q = (sh.o.bmq[x >> 5] >> (x & 31)) & 1u;
            sh.u.sp.q[i] = in_q ? (float)((double)expf(over_T(sh.u.sp.q[i] - qs.m, a.T)) * qs.invZ) : 0.0f;
          }
          q_ready = true;
        }
      }
    }
    if (!q_ready && !lazy) {
      float mx, mn;
      row_maxmin<BLOCK, NC>(v, sh, mx, mn);
      ps.m = mx;
      ps.T = a.T;
      nk = select_kept<BLOCK, NC>(v, V, a.top_k, mx, mn, sh, sh.bm, sh.pre, ps);
      compact_row<BLOCK, NC>(v, V, sh.bm, sh.pre, sh.u.sp.x, sh.u.sp.p);
      __syncthreads();
      ps.invZ = softmax_weights<BLOCK, NC>(sh.u.sp.p, nk, ps.m, a.T, sh);
      for (int i = tid; i < nk; i += BLOCK) sh.u.sp.p[i] = (float)((double)sh.u.sp.p[i] * ps.invZ);
    }
    if (a.stats_out && tid == 0) {
      RowStatsCache c;
      c.m = ps.m; c.T = ps.T; c.tau_v = ps.tau_v; c.tau_x = ps.tau_x; c.all = ps.all ? 1 : 0;
      c.top_k = a.top_k; c.tag = a.stats_tag; c.pad = 0; c.invZ = ps.invZ;
      a.stats_out[(size_t)b * L + j] = c;
    }
    if (a.dbg_p) {
      float4* dst = (float4*)(a.dbg_p + ((size_t)b * L + j) * V);
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int c = tid + i * BLOCK;
        if (c < nchunk) {
          float4 o;
          o.x = ps.prob(v[i].x, 4 * c);
          o.y = ps.prob(v[i].y, 4 * c + 1);
          o.z = ps.prob(v[i].z, 4 * c + 2);
          o.w = ps.prob(v[i].w, 4 * c + 3);
          dst[c] = o;
        }
      }
    }
    __syncthreads();
  }
  auto prow = [&](int ent) -> float { return sh.u.sp.p[ent]; };
  // the compact list for the draws that need it (candidate path: built here,
  // with the draft probabilities when the row has candidates)
  auto need_list = [&]() {
    if (lazy) {
      fast_build_list<BLOCK, NC>(sh, ps, qs, ncand > 0, two, ld.draft);
      lazy = false;
    }
  };

  // ---- sibling rows: bonus draw from the sibling's own output row
  if (!spine) {
    const int sib_d = (j - n_s) / Km1, sib_k = (j - n_s) % Km1 + 2;
    const int sib_tok = a.sib ? a.sib[(size_t)b * trial_stride(a, (size_t)a.D * Km1) + (size_t)sib_d * Km1 + (sib_k - 2)] : -1;
    int tok = -1, stage = 0;
    if (sib_tok < 0 || forced_pos(a, g0 + sib_d)) {
      tok = -1; stage = 0;
    } else if (forced_pos(a, g0 + sib_d + 1)) {
      tok = -1; stage = -1;
    } else {
      const Stream rs(a.seed, kTagBonus, 0, (uint32_t)j, (uint32_t)b, a.step);
      need_list();
      tok = race_compact<BLOCK, NC>(sh, sh, nk, rs, prow);
    }
    if (tid == 0) {
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
  if (!ld.need_p && !a.dbg_p) {  // row-end position: the token is forced
    if (tid == 0) {
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
  if (forced_pos(a, g0 + j)) {  // (debug output requested on a forced row)
    if (tid == 0) {
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

  int out_tok = -1, out_stage = 0;
  if (ncand > 0) {
    const float* draft_row = ld.draft;
    if (q_ready) {
      // computed together with the target row
    } else if (ld.q_cached) {
      // the previous step computed this row's distribution: its statistics,
      // and the draft logits at the target's kept entries (gathered)
      const RowStatsCache c = *ld.q_cached;
      qs.m = c.m; qs.T = c.T; qs.tau_v = c.tau_v; qs.tau_x = c.tau_x; qs.all = c.all != 0; qs.invZ = c.invZ;
      if (!lazy) {
        for (int i = tid; i < nk; i += BLOCK) {
          const int x = (int)sh.u.sp.x[i];
          const float l = draft_row[x];
          sh.u.sp.q[i] = qs.in_set(l, x) ? (float)((double)expf(over_T(l - qs.m, a.T)) * qs.invZ) : 0.0f;
        }
        __syncthreads();
      }
    } else {
    // draft row: selection, then its logits at the kept entries
    if (!PF) load_row<BLOCK, NC>(vq, draft_row, V);
    float qmx, qmn;
    row_maxmin<BLOCK, NC>(vq, sh, qmx, qmn);
    qs.m = qmx;
    qs.T = a.T;
    const int nq = select_kept<BLOCK, NC>(vq, V, a.top_k, qmx, qmn, sh, sh.o.bmq, sh.o.preq, qs);
    // draft logits at the target's kept entries (by target rank) and at its
    // own kept entries (by draft rank, for its normaliser)
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int c = tid + i * BLOCK;
      if (c < nchunk) {
        const int sh4 = 4 * (c & 7);
        const uint32_t wp = sh.bm[c >> 3], wq = sh.o.bmq[c >> 3];
        const uint32_t np = (wp >> sh4) & 15u, nqb = (wq >> sh4) & 15u;
        if (np | nqb) {
          int rp = sh.pre[c >> 3] + __popc(wp & ((1u << sh4) - 1u));
          int rq = sh.o.preq[c >> 3] + __popc(wq & ((1u << sh4) - 1u));
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float l = comp(vq[i], e);
            if ((np >> e) & 1u) sh.u.sp.q[rp++] = l;
            if ((nqb >> e) & 1u) sh.o.qc[rq++] = l;
          }
        }
      }
    }
    __syncthreads();
    qs.invZ = softmax_weights<BLOCK, NC>(sh.o.qc, nq, qs.m, a.T, sh);
    for (int i = tid; i < nk; i += BLOCK) {
      const int x = (int)sh.u.sp.x[i];
      const bool in_q = (sh.o.bmq[x >> 5] >> (x & 31)) & 1u;
      sh.u.sp.q[i] = in_q ? (float)((double)expf(over_T(sh.u.sp.q[i] - qs.m, a.T)) * qs.invZ) : 0.0f;
    }
    __syncthreads();
    }
    auto qrow_c = [&](int ent) -> float { return sh.u.sp.q[ent]; };

    float Qsum = 0.0f;
    float Nf = 1.0f;
    for (int k = 1; k <= ncand; ++k) {
      int x = stg.cand[0];
#pragma unroll
      for (int t = 1; t < 8; ++t) x = (t == k - 1) ? stg.cand[t] : x;
      const float lq = k == 1 ? qcl0 : draft_row[x];
      const float lp = k == 1 ? pcl0 : ld.cur[x];
      const float den = 1.0f - Qsum;
      // at stage 1 the normaliser and the remaining draft mass are 1, so
      // p^(1) and q^(1) are p and q exactly; the weights of the first
      // candidate are those exp((l - max) / T) the selection computed
      const bool first_fast = k == 1 && fast_first;
      const float px = first_fast ? (ps.in_set(lp, x) ? (float)((double)ep0 * ps.invZ) : 0.0f) : ps.prob(lp, x);
      const float qx = (first_fast && two) ? (qs.in_set(lq, x) ? (float)((double)eq0 * qs.invZ) : 0.0f)
                                           : qs.prob(lq, x);
      const float pk = k == 1 ? px : stg.rho(px, qx, x) / Nf;
      const float qk = k == 1 ? qx : (den > 0.0f ? qx / den : 0.0f);
      const float u = k == 1 ? u0 : u01(Stream(a.seed, kTagAcc, (uint32_t)(k - 1), (uint32_t)j, (uint32_t)b, a.step).word(0));
      const bool acc = qk > 0.0f ? (u < pk / qk) : (pk > 0.0f);
      if (acc) {
        out_tok = x;
        out_stage = k;
        break;
      }
      // residual of this stage
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (t == stg.n) { stg.Nf[t] = Nf; stg.den[t] = den; }
      stg.n += 1;
      need_list();
      Qsum = Qsum + qx;
      // the last candidate's residual needs no normaliser (the draw below
      // races its unnormalised weights); it has mass iff one weight is
      // positive, which the draw itself finds out
      if (k == ncand) break;
      double nd = 0.0;
      for (int ent = tid; ent < nk; ent += BLOCK)
        nd += (double)stg.rho(sh.u.sp.p[ent], sh.u.sp.q[ent], (int)sh.u.sp.x[ent]);
      nd = block_sum_d<W>(nd, sh.red_d);
      if (!(nd > 0.0)) {
        stg.n -= 1;  // no residual mass: draw from p^(k) itself
        break;
      }
      Nf = (float)nd;
    }
    if (out_stage == 0) {
      // candidates tried: all of them unless the loop left through the
      // zero-mass exit, in which case that stage was tried too
      const int tried = stg.n + (stg.n < ncand ? 1 : 0);
      const Stream rs(a.seed, kTagRes, (uint32_t)tried, (uint32_t)j, (uint32_t)b, a.step);
      need_list();
      auto draw = [&]() {
        return race_compact<BLOCK, NC>(sh, sh, nk, rs, [&](int ent) -> float {
          return stg.rho(sh.u.sp.p[ent], qrow_c(ent), (int)sh.u.sp.x[ent]);
        });
      };
      out_tok = draw();
      if (out_tok < 0 && stg.n == ncand) {
        // the last residual has no mass (a rounding artefact): draw from
        // p^(ncand) itself, from the same stream
        stg.n -= 1;
        out_tok = draw();
      }
    }
  } else {
    // no draft distribution (appended placeholder) or no valid candidate:
    // a plain draw from p, counted as a rejection
    const Stream rs(a.seed, kTagRes, 0, (uint32_t)j, (uint32_t)b, a.step);
    need_list();
    out_tok = race_compact<BLOCK, NC>(sh, sh, nk, rs, prow);
    out_stage = 0;
  }

  // vanilla SJD: a fresh draw from p replaces the row in the next window
  int fresh = out_tok;
  if (!ac) {
    const Stream rs(a.seed, kTagFresh, 0, (uint32_t)j, (uint32_t)b, a.step);
    need_list();
    fresh = race_compact<BLOCK, NC>(sh, sh, nk, rs, prow);
  }

  // proactive drafting: a small launch (every row resident at once) draws
  // each row's candidates here; otherwise k_verify_pd draws them for the
  // rows the next window drafts at, from the statistics this row leaves
  const bool inl = pd && (a.flags & kFlagPDInline);
  int pds[7];
  if (inl) {
    need_list();
    draft_candidates<BLOCK, NC>(a, sh, nk, ac ? out_tok : fresh, j, b, Km1, pds);
  }
  if (tid == 0) {
    rec[0] = out_tok;
    rec[1] = out_stage;
    rec[9] = fresh;
    put_stats(rec, ps);
    if (inl) {
#pragma unroll
      for (int t = 0; t < 7; ++t)
        if (t < Km1) rec[2 + t] = pds[t];
    }
    if (a.out_rows) {
      int32_t* o = a.out_rows + ((size_t)b * L + j) * 2;
      o[0] = out_tok < 0 ? -1 : out_tok + a.vis_lo;
      o[1] = out_stage;
    }
  }
}

// One workgroup per row (row = trial * L + window row); for 512 threads or
// more the register budget is capped so that two workgroups share a compute
// unit.
template <int BLOCK, int NC, bool PF>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(BLOCK >= 512 ? 4 : 1))) void k_verify_rows(VerifyArgs a) {
  __shared__ VSh<BLOCK, NC> sh;
  const int row = blockIdx.x;
  float4 v[NC];
  if constexpr (PF) {
    // the row's own logits are read before the plan is known (the row lies
    // in the logits buffer whatever the window says; a row that turns out to
    // be unused costs one read)
    load_row<BLOCK, NC>(v, row_logits(a, row), a.V);
    const RowLoad ld = plan_load(a, row);
    float4 vq[NC];
    if (ld.need_q && !ld.q_cached) load_row<BLOCK, NC>(vq, ld.draft, a.V);
    verify_row<BLOCK, NC, true>(a, sh, row, ld, v, vq);
  } else {
    const RowLoad ld = plan_load(a, row);
    verify_row<BLOCK, NC, false>(a, sh, row, ld, v, v);
  }
}

// ------------------------------------------------------------ finalize
__global__ __launch_bounds__(kWave) void k_verify_finalize(VerifyArgs a, FinalizeOut o) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int L = a.L, V = a.V, K = a.K, Km1 = a.K - 1, D = a.D;
  const int32_t* meta = a.in_meta + (size_t)b * trial_stride(a, 4);
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
  // the drafting candidates of depths d < Dn: drawn by the rows themselves
  // (small launches) or afterwards by k_verify_pd
  const bool inl = (a.flags & kFlagPDInline) != 0;
  int32_t* osib = o.out_sib + (size_t)b * o.sib_stride;
  for (int i = lane; i < D * Km1; i += kWave) {
    const int d = i / Km1, k = i % Km1;
    int t = -1;
    if (inl && d < Dn) {
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

// ------------------------------------------------------------ drafting
// One workgroup per (trial, depth d): after finalize, the next window's
// siblings at depth d < D' come from row n_c + d of this step (proactive
// drafting, Sec. 4.1; Alg. 1 drafts only after a rejection). The row's kept
// set is rebuilt from its logits and the statistics its row kernel left in
// its record (the same threshold, maximum and normaliser, so the same
// probabilities and ranks), and the K - 1 candidates are drawn without
// replacement excluding the token the row carries forward. Only the rows
// the next window drafts at pay for the draws.
// Shared memory of the drafting kernel: the kept set, its prefix counts and
// the compact list (tokens and probabilities) only, about a quarter of the
// row kernel's, so four workgroups share a compute unit instead of two.
template <int BLOCK, int NC>
struct PdSh {
  static constexpr int W = BLOCK / kWave;
  static constexpr int NW = BLOCK * NC / 8;  // bitmap words (32 entries each)
  struct List {
    uint16_t x[kKcap];
    float p[kKcap];
  };
  uint32_t bm[NW];
  int32_t pre[NW];
  union {
    List sp;
  } u;
  uint64_t pd_w[W * 8];
  int pd_o[8];
  int red_i[2 * W];
  int ncand[2];
};

template <int BLOCK, int NC>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(BLOCK >= 512 ? 4 : 1))) void k_verify_pd(
    VerifyArgs a, FinalizeOut o) {
  __shared__ PdSh<BLOCK, NC> sh;
  constexpr int W = BLOCK / kWave;
  const int tid = threadIdx.x;
  const int b = blockIdx.x / a.D, d = blockIdx.x % a.D;
  const int L = a.L, Km1 = a.K - 1;
  const int32_t* om = o.out_meta + (size_t)b * o.meta_stride;
  const int n_c = om[0], Dn = om[2];
  if (n_c < 0 || d >= Dn) return;  // (invalid trial, or no drafting at this depth)
  const int jj = n_c + d;
  const int32_t* rec = a.rec + ((size_t)b * L + jj) * kRecInts;
  if (rec[1] == -1) return;  // row end: no siblings
  const int excl = (a.flags & kFlagAC) ? rec[0] : rec[9];
  const RowStats st = get_stats(rec, a.T);
  float4 v[NC];
  load_row<BLOCK, NC>(v, row_logits(a, b * L + jj), a.V);
  bitmap_from_tau<BLOCK, NC>(v, a.V, st, sh.bm);
  __syncthreads();
  constexpr int NW = PdSh<BLOCK, NC>::NW;
  constexpr int WPT = NW / BLOCK > 0 ? NW / BLOCK : 1;
  int cnt[WPT];
  int s0 = 0;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    cnt[i] = wi < NW ? __popc(sh.bm[wi]) : 0;
    s0 += cnt[i];
  }
  int run = block_excl_scan<W>(s0, sh.red_i);
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int wi = tid * WPT + i;
    if (wi < NW) sh.pre[wi] = run;
    run += cnt[i];
  }
  if (tid == BLOCK - 1) sh.ncand[0] = run;
  __syncthreads();
  const int nk = sh.ncand[0];
  compact_row<BLOCK, NC>(v, a.V, sh.bm, sh.pre, sh.u.sp.x, sh.u.sp.p);
  __syncthreads();
  for (int i = tid; i < nk; i += BLOCK) sh.u.sp.p[i] = (float)((double)expf(over_T(sh.u.sp.p[i] - st.m, a.T)) * st.invZ);
  __syncthreads();
  int pds[7];
  draft_candidates<BLOCK, NC>(a, sh, nk, excl, jj, b, Km1, pds);
  if (tid < Km1) {
    int y = -1;
#pragma unroll
    for (int t = 0; t < 7; ++t) y = t == tid ? pds[t] : y;
    o.out_sib[(size_t)b * o.sib_stride + (size_t)d * Km1 + tid] = y < 0 ? -1 : y + a.vis_lo;
  }
}

// ------------------------------------------------------------ no-alloc scratch
// The per-row records of sjd_verify_noalloc live in a static device array
// (every device the library runs on holds its own copy until the process
// ends). Host code never passes the array's name to a kernel: its device
// address is looked up per device with hipGetSymbolAddress and kept.
// (plus 64 words: the SJD_CHECK_FINITE count word follows the records)
static __device__ __align__(256) int32_t scratch[(size_t)SJD_VERIFY_NOALLOC_MAX_ROWS * kRecInts + 64];

hipError_t noalloc_scratch(int32_t** out) {
  static std::mutex mu;
  static std::vector<int32_t*> addr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  if ((int)addr.size() <= dev) addr.resize(dev + 1, nullptr);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = (int32_t*)p;
  }
  *out = addr[dev];
  return hipSuccess;
}

// ------------------------------------------------------------ launch
hipError_t launch_verify(const VerifyArgs& a0, const FinalizeOut& o, hipStream_t s) {
  const long rows = (long)a0.B * a0.L;
  if (rows < 1 || rows > 0x7FFFFFFFL) return hipErrorInvalidValue;
  // a launch whose rows are all resident at once (two workgroups per compute
  // unit) draws the drafting candidates in the row kernel: a second kernel
  // would only add its latency
  VerifyArgs a = a0;
  const bool pd = (a.flags & kFlagPD) && a.K >= 2 && a.D >= 1;
  if (pd && rows <= kPdInlineRows) a.flags |= kFlagPDInline;
  const dim3 grid((unsigned)rows);
  if (a.V <= 4096) hipLaunchKernelGGL((k_verify_rows<256, 4, true>), grid, dim3(256), 0, s, a);
  else if (a.V <= 16384) hipLaunchKernelGGL((k_verify_rows<512, 8, true>), grid, dim3(512), 0, s, a);
  else if (a.V <= 32768) hipLaunchKernelGGL((k_verify_rows<1024, 8, true>), grid, dim3(1024), 0, s, a);
  else if (a.V <= 65536) hipLaunchKernelGGL((k_verify_rows<1024, 16, false>), grid, dim3(1024), 0, s, a);
  else return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_verify_finalize, dim3(a.B), dim3(kWave), 0, s, a, o);
  e = hipGetLastError();
  if (e != hipSuccess || !pd || (a.flags & kFlagPDInline)) return e;
  const dim3 gpd((unsigned)((long)a.B * a.D));
  if (a.V <= 4096) hipLaunchKernelGGL((k_verify_pd<256, 4>), gpd, dim3(256), 0, s, a, o);
  else if (a.V <= 16384) hipLaunchKernelGGL((k_verify_pd<512, 8>), gpd, dim3(512), 0, s, a, o);
  else if (a.V <= 32768) hipLaunchKernelGGL((k_verify_pd<1024, 8>), gpd, dim3(1024), 0, s, a, o);
  else hipLaunchKernelGGL((k_verify_pd<1024, 16>), gpd, dim3(1024), 0, s, a, o);
  return hipGetLastError();
}

}  // namespace sjd
