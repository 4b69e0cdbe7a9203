// Window attention: M <= 64 query slots of one head against the cached keys
// and values plus the window's own (tree-masked) keys, on bf16 MFMA.
//
// Layout choices (gfx950, wave64, v_mfma_f32_32x32x16_bf16):
//  - scores are formed transposed, S^T = K . Q^T (rows = keys, columns =
//    slots), so each lane owns one slot: the max, sum and output scaling of
//    the softmax are lane-local (plus one exchange between the two lane
//    halves);
//  - the key rows fed to MFMA row i are key swap23(i); then the score
//    registers of a lane hold 16 keys in the order that O^T = V^T . P^T
//    needs as its B operand, so P never leaves registers;
//  - the caches are tiled in exactly these operand orders (forward.h), so
//    every key or value load is one contiguous 1 KB per wave;
//  - a workgroup handles kAttnChunk = 128 keys of one head for 32 query slots
//    (grid z: slots 0-31, 32-63), 32 keys per wave; the
//    four waves merge in LDS and one partial (unnormalised output, max, sum)
//    per workgroup is combined across chunks by a second kernel;
//  - each wave issues its q chunk, then all of its key and value loads before
//    any arithmetic (the loads are the critical path); q is shared by the
//    four waves through LDS (the same LDS later holds the merge).
// (One wave per workgroup with no merge balances better across compute
// units but writes four times the partials; measured slower.)
// Scores use exp2 with the scale folded into log2(e) / sqrt(hd).
// Precision: q, the cached keys and values, and P are each carried as a
// pair of bf16 values (hi + lo); every product is formed as hi*hi + hi*lo +
// lo*hi on MFMA (the lo*lo term is below fp32 accumulation noise).
#include "device.h"
#include "forward.h"

namespace sjd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

SJD_DEV bf16x8 to_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8, u); }

template <int HD>
struct AttnSmem {
  union {
    uint4 q[2][HD / 16][kWave];  // Q^T operand (hi, lo) in register order, loaded once per workgroup
    float o[4][32][HD + 1];      // merge: [wave][slot][dim], padded against bank conflicts
  };
  float m[4][32];
  float l[4][32];
};

template <int HD>
__global__ __launch_bounds__(256) void k_attn_partial(AttnArgs a) {
  constexpr int NQ = HD / 16;  // MFMAs per 32-key block for the scores
  constexpr int ND = HD / 32;  // 32-dim output blocks
  static_assert(kAttnChunk == 4 * 32, "one 32-key block per wave");
  __shared__ AttnSmem<HD> sm;
  const int h = blockIdx.x, sp = blockIdx.y;
  // multi-stream windows: slot block z is stream z (its own cache and
  // positions, L slots each); otherwise the M slots are one stream
  const bool two = a.st.mode != kStreamsOne;
  const int z = blockIdx.z;
  const int n = stream_rows(a.st, a.n_dev ? *a.n_dev : a.n_host, z);
  const int Ms = two ? a.st.L : a.M, nk = n + Ms;
  const int kbeg = sp * kAttnChunk;
  if (kbeg >= nk) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, r32 = lane & 31, half = lane >> 5;
  const int kvh = h / (a.H / a.Hkv);
  const int zs = blockIdx.z * 32;  // this workgroup's 32 query slots start here
  const int slot = r32;            // local slot (MFMA column)
  const int gslot = zs + slot;
  const bool slot_ok = two ? slot < Ms : gslot < Ms;
  const size_t so = two ? (size_t)z * a.sstride : 0;
  const uint16_t* kc = a.kc + so;
  const uint16_t* kc_lo = a.kc_lo + so;
  const uint16_t* vt = a.vt + so;
  const uint16_t* vt_lo = a.vt_lo + so;
  const int kb = kbeg + wave * 32;  // this wave's key block
  const bool has = kb < nk;
  const size_t tofs = (size_t)kvh * a.cap * HD + (size_t)kb * HD + (size_t)lane * 8;

  // q first (small, cache-resident; the four waves share it through LDS),
  // then the key and value tiles (the long dependencies)
  uint4 qs[2][(NQ + 3) / 4];
  {
    const size_t qo = (size_t)(slot_ok ? gslot : 0) * a.H * HD + (size_t)h * HD + half * (HD / 2);
    const uint4* qp = (const uint4*)(a.q + qo);
    const uint4* qpl = (const uint4*)(a.q_lo + qo);
#pragma unroll
    for (int i = 0; i < (NQ + 3) / 4; ++i) {
      const int t = wave + 4 * i;
      qs[0][i] = (slot_ok && t < NQ) ? qp[t] : make_uint4(0, 0, 0, 0);
      qs[1][i] = (slot_ok && t < NQ) ? qpl[t] : make_uint4(0, 0, 0, 0);
    }
  }
  uint4 kh[NQ], kl[NQ], vh[ND][2], vl[ND][2];
  if (has) {
    const uint4* kp = (const uint4*)(kc + tofs);
    const uint4* kpl = (const uint4*)(kc_lo + tofs);
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      kh[t] = kp[t * 64];
      kl[t] = kpl[t * 64];
    }
    const uint4* vp = (const uint4*)(vt + tofs);
    const uint4* vpl = (const uint4*)(vt_lo + tofs);
#pragma unroll
    for (int d = 0; d < ND; ++d)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        vh[d][jj] = vp[(d * 2 + jj) * 64];
        vl[d][jj] = vpl[(d * 2 + jj) * 64];
      }
  }
  // Q^T operand: lane (slot, half) holds dims half*HD/2 + 8t + e of its
  // slot; wave w staged chunks t = w, w + 4, ...
#pragma unroll
  for (int i = 0; i < (NQ + 3) / 4; ++i) {
    const int t = wave + 4 * i;
    if (t < NQ) {
      sm.q[0][t][lane] = qs[0][i];
      sm.q[1][t][lane] = qs[1][i];
    }
  }
  __syncthreads();

  f32x16 o[ND];
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.0f;
  float m_w = -INFINITY, l_w = 0.0f;
  if (has) {
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      const bf16x8 khb = to_bf16x8(kh[t]), klb = to_bf16x8(kl[t]);
      const bf16x8 qh = to_bf16x8(sm.q[0][t][lane]), ql = to_bf16x8(sm.q[1][t][lane]);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(khb, qh, s, 0, 0, 0);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(khb, ql, s, 0, 0, 0);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(klb, qh, s, 0, 0, 0);
    }
    // mask (register r = 8jj + e holds key kb + 16jj + 8half + e): cached
    // keys are visible to every slot, window keys by the ancestor mask
    if (kb + 32 <= n) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = slot_ok ? s[r] * a.scale : -INFINITY;
    } else {
      const uint64_t anc = slot_ok ? a.win->anc[gslot] : 0ull;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb + 16 * (r >> 3) + 8 * half + (r & 7);
        bool vis = slot_ok && key < nk;
        if (vis && key >= n) vis = (anc >> (key - n)) & 1ull;
        s[r] = vis ? s[r] * a.scale : -INFINITY;
      }
    }
    float mloc = s[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mloc = fmaxf(mloc, s[r]);
    m_w = fmaxf(mloc, __shfl_xor(mloc, 32, kWave));
    float lsum = 0.0f;
    if (m_w != -INFINITY) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = exp2f(s[r] - m_w);
        lsum += s[r];
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
    }
    l_w = lsum + __shfl_xor(lsum, 32, kWave);
    // P^T operand (hi / lo bf16; P is finite, in [0, 1]) and O^T = V^T . P^T
    uint4 pb[2], pbl[2];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      uint32_t w[4], wl[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint16_t h0, l0, h1, l1;
        split_bf16_finite(s[8 * jj + 2 * e], h0, l0);
        split_bf16_finite(s[8 * jj + 2 * e + 1], h1, l1);
        w[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        wl[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
      }
      pb[jj] = make_uint4(w[0], w[1], w[2], w[3]);
      pbl[jj] = make_uint4(wl[0], wl[1], wl[2], wl[3]);
    }
#pragma unroll
    for (int d = 0; d < ND; ++d)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const bf16x8 vhb = to_bf16x8(vh[d][jj]), vlb = to_bf16x8(vl[d][jj]);
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vhb, to_bf16x8(pb[jj]), o[d], 0, 0, 0);
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vhb, to_bf16x8(pbl[jj]), o[d], 0, 0, 0);
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vlb, to_bf16x8(pb[jj]), o[d], 0, 0, 0);
      }
  }

  // ---- merge the four waves (the merge buffer overlays q: wait for every
  // wave's scores first). Output register r of block d holds dim
  // d*32 + 8(r/4) + 4half + r%4 of this lane's slot
  __syncthreads();
#pragma unroll
  for (int d = 0; d < ND; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) sm.o[wave][slot][d * 32 + 8 * (r >> 2) + 4 * half + (r & 3)] = o[d][r];
  if (half == 0) {
    sm.m[wave][slot] = m_w;
    sm.l[wave][slot] = l_w;
  }
  __syncthreads();
  // thread -> (slot, HD/8 consecutive dims)
  constexpr int DPT = HD / 8;
  const int sl = threadIdx.x >> 3, d0 = (threadIdx.x & 7) * DPT;
  float mx = sm.m[0][sl];
#pragma unroll
  for (int w = 1; w < 4; ++w) mx = fmaxf(mx, sm.m[w][sl]);
  float f[4], ls = 0.0f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    f[w] = mx == -INFINITY ? 0.0f : exp2f(sm.m[w][sl] - mx);
    ls += sm.l[w][sl] * f[w];
  }
  float* wo = a.ws_o + (((size_t)h * a.nsplit_max + sp) * kWinRows + zs + sl) * HD + d0;
#pragma unroll
  for (int i = 0; i < DPT; i += 4) {
    float4 v;
    v.x = sm.o[0][sl][d0 + i] * f[0] + sm.o[1][sl][d0 + i] * f[1] + sm.o[2][sl][d0 + i] * f[2] +
          sm.o[3][sl][d0 + i] * f[3];
    v.y = sm.o[0][sl][d0 + i + 1] * f[0] + sm.o[1][sl][d0 + i + 1] * f[1] + sm.o[2][sl][d0 + i + 1] * f[2] +
          sm.o[3][sl][d0 + i + 1] * f[3];
    v.z = sm.o[0][sl][d0 + i + 2] * f[0] + sm.o[1][sl][d0 + i + 2] * f[1] + sm.o[2][sl][d0 + i + 2] * f[2] +
          sm.o[3][sl][d0 + i + 2] * f[3];
    v.w = sm.o[0][sl][d0 + i + 3] * f[0] + sm.o[1][sl][d0 + i + 3] * f[1] + sm.o[2][sl][d0 + i + 3] * f[2] +
          sm.o[3][sl][d0 + i + 3] * f[3];
    *(float4*)(wo + i) = v;
  }
  if ((threadIdx.x & 7) == 0) {
    float* wml = a.ws_ml + ((size_t)h * a.nsplit_max + sp) * kWinRows * 2 + (size_t)(zs + sl) * 2;
    wml[0] = mx;
    wml[1] = ls;
  }
}

// Variant for 128-dim heads (four 32-dim output blocks, one per wave): the
// waves exchange probabilities instead of outputs. Each wave scores its own
// 32 keys as above, writes its P (hi / lo bf16, 4 KB) and softmax statistics
// to LDS, and then forms the output of its own 32 dims over all 128 keys of
// the chunk, loading those dims' value tiles of all four key blocks (the same
// bytes as its own keys' full rows, still contiguous 1 KB loads). This
// replaces a 64 KB fp32 output exchange and its reduction with a 16 KB
// probability exchange; the partial then leaves in four independent 4 KB
// slices. A workgroup serves every query head of its key / value head
// (grouped-query attention) from the same registers: the tiles are read
// once per group instead of once per query head.
struct AttnPxSmem {
  uint4 q[2][8][kWave];     // Q^T operand (hi, lo), 128 dims
  uint4 p[4][2][2][kWave];  // [key block][16-key half][hi / lo][lane]: P^T operand
  float m[4][32];
  float l[4][32];
};

// The query heads of a key / value head (grouped-query attention) are dealt
// to a.qparts workgroups, blockIdx.x = kv head + Hkv * part. Workgroups go to
// the XCDs round-robin by launch index, so with Hkv a multiple of the XCD
// count every part of a head (and every chunk of it) runs on one XCD: the
// head's key and value tiles come from HBM once and from that XCD's L2 for
// the other parts. MULTI: a workgroup takes several query heads, one after
// another, the next head's q read while the current one computes.
template <bool MULTI>
__global__ __launch_bounds__(256) void k_attn_partial_px(AttnArgs a) {
  constexpr int HD = 128, NQ = HD / 16;
  static_assert(kAttnChunk == 4 * 32, "one 32-key block per wave");
  __shared__ AttnPxSmem sm;
  const int kvh = (int)blockIdx.x % a.Hkv, part = (int)blockIdx.x / a.Hkv, sp = blockIdx.y;
  const int G = a.H / a.Hkv / a.qparts;  // query heads of this workgroup
  const int g0 = part * G;               // the first of them, within the key / value head's group
  const bool two = a.st.mode != kStreamsOne;
  const int z = blockIdx.z;
  const int n = stream_rows(a.st, a.n_dev ? *a.n_dev : a.n_host, z);
  const int Ms = two ? a.st.L : a.M, nk = n + Ms;
  const int kbeg = sp * kAttnChunk;
  if (kbeg >= nk) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, half = lane >> 5;
  const int zs = blockIdx.z * 32;
  const int slot = lane & 31;
  const int gslot = zs + slot;
  const bool slot_ok = two ? slot < Ms : gslot < Ms;
  const size_t hbase = (size_t)kvh * a.cap * HD + (two ? (size_t)z * a.sstride : 0);
  const int kb = kbeg + wave * 32;  // this wave's key block
  const bool has = kb < nk;

  // the first query head's q chunks go first (small, cache-resident; vector
  // loads return in order, so a q load issued after the tiles would wait for
  // all of them), then the key / value tiles, which stay in registers for
  // every query head of the group
  auto load_q = [&](int h, uint4 (&qr)[2][2]) {
    const size_t qo = (size_t)(slot_ok ? gslot : 0) * a.H * HD + (size_t)h * HD + half * (HD / 2);
    const uint4* qp = (const uint4*)(a.q + qo);
    const uint4* qpl = (const uint4*)(a.q_lo + qo);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int t = wave + 4 * i;
      qr[0][i] = slot_ok ? qp[t] : make_uint4(0, 0, 0, 0);
      qr[1][i] = slot_ok ? qpl[t] : make_uint4(0, 0, 0, 0);
    }
  };
  const int hq0 = kvh * (a.H / a.Hkv) + g0;  // this workgroup's first query head
  uint4 qs[2][2];
  load_q(hq0, qs);
  uint4 kh[NQ], kl[NQ], vh[4][2], vl[4][2];
  if (has) {
    const uint4* kp = (const uint4*)(a.kc + hbase + (size_t)kb * HD + (size_t)lane * 8);
    const uint4* kpl = (const uint4*)(a.kc_lo + hbase + (size_t)kb * HD + (size_t)lane * 8);
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      kh[t] = kp[t * 64];
      kl[t] = kpl[t * 64];
    }
  }
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int kbw = kbeg + w * 32;
    const uint4* vp = (const uint4*)(a.vt + hbase + (size_t)kbw * HD + (size_t)lane * 8);
    const uint4* vpl = (const uint4*)(a.vt_lo + hbase + (size_t)kbw * HD + (size_t)lane * 8);
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {  // absent blocks: zeros (their P is zero; 0 * garbage could be NaN)
      vh[w][jj] = kbw < nk ? vp[(wave * 2 + jj) * 64] : make_uint4(0, 0, 0, 0);
      vl[w][jj] = kbw < nk ? vpl[(wave * 2 + jj) * 64] : make_uint4(0, 0, 0, 0);
    }
  }
  // mask of this wave's keys for this lane's slot (the same for every head)
  uint32_t vis = 0;
  if (has && slot_ok) {
    const uint64_t anc = kb + 32 <= n ? 0ull : a.win->anc[gslot];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = kb + 16 * (r >> 3) + 8 * half + (r & 7);
      bool v = key < nk;
      if (v && key >= n) v = (anc >> (key - n)) & 1ull;
      vis |= (v ? 1u : 0u) << r;
    }
  }

  for (int g = 0; g < G; ++g) {
    const int h = hq0 + g;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      sm.q[0][wave + 4 * i][lane] = qs[0][i];
      sm.q[1][wave + 4 * i][lane] = qs[1][i];
    }
    __syncthreads();  // (also: every wave is done with the previous head's P)
    // several heads: the next head's q is read while this one computes (the
    // last re-reads its own: an unconditional load keeps the wait counts
    // exact)
    if constexpr (MULTI) load_q(g + 1 < G ? h + 1 : h, qs);

    float m_w = -INFINITY, l_w = 0.0f;
    uint4 pb[2] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)}, pbl[2] = {pb[0], pb[1]};
    if (has) {
      f32x16 s;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
      for (int t = 0; t < NQ; ++t) {
        const bf16x8 khb = to_bf16x8(kh[t]), klb = to_bf16x8(kl[t]);
        const bf16x8 qh = to_bf16x8(sm.q[0][t][lane]), ql = to_bf16x8(sm.q[1][t][lane]);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(khb, qh, s, 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(khb, ql, s, 0, 0, 0);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(klb, qh, s, 0, 0, 0);
      }
      // mask (register r = 8jj + e holds key kb + 16jj + 8half + e)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = (vis >> r) & 1u ? s[r] * a.scale : -INFINITY;
      float mloc = s[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mloc = fmaxf(mloc, s[r]);
      m_w = fmaxf(mloc, __shfl_xor(mloc, 32, kWave));
      float lsum = 0.0f;
      if (m_w != -INFINITY) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[r] = exp2f(s[r] - m_w);
          lsum += s[r];
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.0f;
      }
      l_w = lsum + __shfl_xor(lsum, 32, kWave);
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        uint32_t w[4], wl[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint16_t h0, l0, h1, l1;
          split_bf16_finite(s[8 * jj + 2 * e], h0, l0);
          split_bf16_finite(s[8 * jj + 2 * e + 1], h1, l1);
          w[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
          wl[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        pb[jj] = make_uint4(w[0], w[1], w[2], w[3]);
        pbl[jj] = make_uint4(wl[0], wl[1], wl[2], wl[3]);
      }
    }
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      sm.p[wave][jj][0][lane] = pb[jj];
      sm.p[wave][jj][1][lane] = pbl[jj];
    }
    if (half == 0) {
      sm.m[wave][slot] = m_w;
      sm.l[wave][slot] = l_w;
    }
    __syncthreads();

    // O^T (this wave's 32 dims x 32 slots) = sum over key blocks w of
    // 2^(m_w - m) V_w^T . P_w^T
    float mw[4], mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      mw[w] = sm.m[w][slot];
      mx = fmaxf(mx, mw[w]);
    }
    f32x16 o;
#pragma unroll
    for (int r = 0; r < 16; ++r) o[r] = 0.0f;
    float ls = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = mx == -INFINITY ? 0.0f : exp2f(mw[w] - mx);
      ls += sm.l[w][slot] * f;
      f32x16 t;
#pragma unroll
      for (int r = 0; r < 16; ++r) t[r] = 0.0f;
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const bf16x8 vhb = to_bf16x8(vh[w][jj]), vlb = to_bf16x8(vl[w][jj]);
        const bf16x8 ph = to_bf16x8(sm.p[w][jj][0][lane]), pl = to_bf16x8(sm.p[w][jj][1][lane]);
        t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vhb, ph, t, 0, 0, 0);
        t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vhb, pl, t, 0, 0, 0);
        t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vlb, ph, t, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) o[r] += f * t[r];
    }
    // register r of lane (slot, half): dim 32 wave + 8(r/4) + 4 half + r%4
    float* wo = a.ws_o + (((size_t)h * a.nsplit_max + sp) * kWinRows + zs + slot) * HD + wave * 32 + 4 * half;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4)
      *(float4*)(wo + 8 * q4) = make_float4(o[4 * q4], o[4 * q4 + 1], o[4 * q4 + 2], o[4 * q4 + 3]);
    if (wave == 0 && half == 0) {
      float* wml = a.ws_ml + ((size_t)h * a.nsplit_max + sp) * kWinRows * 2 + (size_t)(zs + slot) * 2;
      wml[0] = mx;
      wml[1] = ls;
    }
  }
}

// out[slot][h*hd + dim] = sum_s o_s 2^(m_s - m) / sum_s l_s 2^(m_s - m).
// grid (H, HD / 32, slot halves), block 256: thread -> (slot, 4 consecutive dims).
// The partials were written by workgroups on every XCD (far-memory round
// trips), so the splits are taken in groups of kCombGroup whose loads are all
// in flight at once; groups are merged with a running maximum.
constexpr int kCombGroup = 16;
template <int HD>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  const int h = blockIdx.x, t = threadIdx.x;
  const int slot = blockIdx.z * 32 + (t >> 3), dim0 = blockIdx.y * 32 + (t & 7) * 4;
  if (slot >= a.M) return;
  const size_t oo = (size_t)slot * a.ldo + (size_t)h * HD + dim0;
  const bool two = a.st.mode != kStreamsOne;
  if (two && (slot & 31) >= a.st.L) {  // padding row of a multi-stream window: finite zeros
    *(ushort4*)(a.out + oo) = make_ushort4(0, 0, 0, 0);
    *(ushort4*)(a.out_lo + oo) = make_ushort4(0, 0, 0, 0);
    return;
  }
  const int n = stream_rows(a.st, a.n_dev ? *a.n_dev : a.n_host, slot >> 5);
  const int nk = n + (two ? a.st.L : a.M);
  const int ns = (nk + kAttnChunk - 1) / kAttnChunk;
  const float* wml = a.ws_ml + (size_t)h * a.nsplit_max * kWinRows * 2 + slot * 2;
  const float* wo = a.ws_o + ((size_t)h * a.nsplit_max * kWinRows + slot) * HD + dim0;
  float mx = -INFINITY, ls = 0.0f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < ns; s0 += kCombGroup) {
    float2 ml[kCombGroup];
    float4 v[kCombGroup];
#pragma unroll
    for (int i = 0; i < kCombGroup; ++i) {
      const int sx = s0 + i < ns ? s0 + i : ns - 1;
      ml[i] = *(const float2*)(wml + (size_t)sx * kWinRows * 2);
      v[i] = *(const float4*)(wo + (size_t)sx * kWinRows * HD);
    }
    float gm = mx;
#pragma unroll
    for (int i = 0; i < kCombGroup; ++i)
      if (s0 + i < ns) gm = fmaxf(gm, ml[i].x);
    if (gm != mx && mx != -INFINITY) {  // rescale what the earlier groups summed
      const float r = exp2f(mx - gm);
      ls *= r;
      acc.x *= r;
      acc.y *= r;
      acc.z *= r;
      acc.w *= r;
    }
    mx = gm;
#pragma unroll
    for (int i = 0; i < kCombGroup; ++i)
      if (s0 + i < ns) {
        const float f = ml[i].x == -INFINITY ? 0.0f : exp2f(ml[i].x - mx);
        ls += ml[i].y * f;
        acc.x += v[i].x * f;
        acc.y += v[i].y * f;
        acc.z += v[i].z * f;
        acc.w += v[i].w * f;
      }
  }
  ushort4 hi, lo;
  split_bf16(acc.x / ls, hi.x, lo.x);
  split_bf16(acc.y / ls, hi.y, lo.y);
  split_bf16(acc.z / ls, hi.z, lo.z);
  split_bf16(acc.w / ls, hi.w, lo.w);
  *(ushort4*)(a.out + oo) = hi;
  *(ushort4*)(a.out_lo + oo) = lo;
}

hipError_t launch_attention(const AttnArgs& a, int hd, hipStream_t s) {
  if (a.M < 1 || a.M > (a.st.mode == kStreamsOne ? 64 : 32 * kMaxStreams)) return hipErrorInvalidValue;
  const unsigned zh = (unsigned)(a.M + 31) / 32;  // 32-slot blocks
  const dim3 g1(a.H, a.nsplit_max, zh), g2(a.H, hd / 32, zh);
  if (hd == 128) {
    // one workgroup per key / value head: its tiles are read once for the
    // whole group of query heads that share them
    const int G = a.H / a.Hkv;
    if (a.qparts < 1 || G % a.qparts) return hipErrorInvalidValue;
    const dim3 gp((unsigned)(a.Hkv * a.qparts), a.nsplit_max, zh);
    if (G / a.qparts > 1) hipLaunchKernelGGL(k_attn_partial_px<true>, gp, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_attn_partial_px<false>, gp, dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_attn_combine<128>, g2, dim3(256), 0, s, a);
  } else if (hd == 64) {
    hipLaunchKernelGGL(k_attn_partial<64>, g1, dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_attn_combine<64>, g2, dim3(256), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sjd
