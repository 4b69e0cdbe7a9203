// Skinny bf16 GEMM for the window forward: C[M x N] = A[M x K] . W[N x K]^T
// with M <= 128 window slots (up to four streams of 32), on gfx950 MFMA
// (v_mfma_f32_32x32x16_bf16).
//
// The window forward is bound by streaming the weights from HBM (2 flop per
// weight byte per slot: 64 flop/B at M = 32, far below the MFMA ridge), so
// the kernel is laid out for the weight stream:
//  - weights are pre-tiled (see forward.h): a wave reads one 32-row x 64-k
//    tile per k-step as four contiguous 1 KB loads, the next k-step in flight,
//    and the column blocks' tiles of a k-step form one contiguous stripe;
//  - the activation tile of a k-step (32 rows x 64 k, hi and lo planes, 8 KB
//    per 32 rows) is staged once per workgroup into LDS (double buffered) and
//    shared by its NW waves (4 or 8), each of which owns a different
//    32-column block. Loading A per wave from L2 instead costs twice the
//    weight bytes again and halves the achieved weight bandwidth; eight
//    column blocks per workgroup halve the activation loads per weight byte
//    again, which 64-row windows need most (their QKV, gate/up and LM-head
//    GEMMs ran 17-27% faster);
//  - the contraction index is permuted identically in A and W (any
//    permutation of k leaves the sum unchanged), so both operands load as
//    16-byte chunks straight into the MFMA register layout;
//  - the K range is split across S workgroups that write separate fp32
//    partial planes; the kernel that consumes the result sums the planes in a
//    fixed order (deterministic, and no device-scope fence, which on this
//    part would write back and invalidate the L2).
// Activations arrive as two bf16 planes (hi + lo, about 16 significant
// bits): the weights are exact bf16, so two MFMAs per tile recover an
// fp32-class product at no HBM cost (the MFMA units are otherwise idle).
// Epilogue: optional per-row RMS scale (the normalisation of a preceding
// RMSNorm, whose gain is already folded into A), then store fp32 to plane sp;
// for a guided head, the guidance combine of row pairs (64b + m, 64b + 32 + m).
#include "device.h"
#include "forward.h"

namespace sjd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// column blocks (= waves) per workgroup: 4, or 8 when GemmArgs::wide
constexpr int kGWaves = 4;
constexpr int kGWavesWide = 8;
// k-steps held per wave (the current one plus one in flight): deeper rings
// help a lone workgroup but lose once every compute unit holds several
constexpr int kRingDepth = 2;
constexpr int kRingDeep = 4;
// RMSNorm chunk sums held in registers (d <= 4096; larger d reads the rest late)
constexpr int kSsRegs = 16;

SJD_DEV bf16x8 as_bf16x8(const u32x4& u) { return __builtin_bit_cast(bf16x8, u); }

template <int MT>
struct GemmSmem {
  u32x4 a[2][2][MT][4][kWave];  // [buffer][hi / lo][row tile][16-byte chunk][lane]: A tiles in MFMA operand order
  float inv[32 * MT];
};

// The main loop is straight-line code: vector loads return in issue order
// and the wait before a use covers everything issued earlier, so no load is
// ever consumed in the step that issued it, loads are never conditional
// (a branch makes the compiler's wait counts conservative), and within a
// step the activation chunk is issued before the weight tile. The step count
// is padded to a multiple of the ring: padded steps reload the last real
// tile and stage a zero activation tile, so they add nothing.
// MT = 32-row tiles of A (M <= 32 MT).
// Workgroups are dealt to the XCDs round-robin by launch index (index i runs
// on XCD i % kXcds). The grid is one-dimensional, and (column group, K
// split) is chosen so that each XCD runs a contiguous run of the
// split-major order: its workgroups share few K splits, so each XCD pulls
// few activation tiles into its own L2 (with the plain 2D order, every XCD
// ran every split and fetched the whole activation).
constexpr int kXcds = 8;
SJD_DEV void gemm_tile_of(int id, int groups, int splits, int& group, int& split) {
  const int total = groups * splits;
  const int q = total / kXcds, r = total % kXcds;
  const int xcd = id % kXcds, j = id / kXcds;
  const int lin = xcd < r ? xcd * (q + 1) + j : r * (q + 1) + (xcd - r) * q + j;
  split = lin / groups;
  group = lin % groups;
}

template <int kRing, int MT, int NW>
__global__ __launch_bounds__(NW * kWave) void k_gemm(GemmArgs g) {
  __shared__ GemmSmem<MT> sm;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int r32 = lane & 31, half = lane >> 5;
  const int T = g.K / 64, nblk = g.N / 32;
  const int groups = (nblk + NW - 1) / NW;
  int group, sp;
  gemm_tile_of((int)blockIdx.x, groups, g.S, group, sp);
  const int nb = group * NW + wave;  // this wave's 32-column block
  const bool active = nb < nblk;
  const int st0 = (int)((long)T * sp / g.S), st1 = (int)((long)T * (sp + 1) / g.S);
  const int n = st1 - st0;
  const int npad = (n + kRing - 1) / kRing * kRing;

  // fused RMSNorm: row scale from the chunk sums of squares. The loads go
  // into registers ahead of the weight stream and are summed after it (a sum
  // here would wait for them before the first weight load is issued).
  const bool has_ss = g.ss != nullptr && (int)threadIdx.x < 32 * MT;
  const float* ssr = has_ss ? g.ss + (size_t)((int)threadIdx.x < g.M ? threadIdx.x : 0) * g.ss_n : nullptr;
  float ssv[kSsRegs];
  if (has_ss)
#pragma unroll
    for (int c = 0; c < kSsRegs; ++c) ssv[c] = ssr[c < g.ss_n ? c : 0];

  // element (row mt*32 + r32, k = kb*64 + half*32 + i*8 + e) of a tile sits
  // in chunk i of lane r32 + 32*half of row tile mt. The 8 MT staged chunks
  // of a k-step (plane, row tile, chunk) are numbered q = (plane MT + mt) 4
  // + chunk, and wave w stages q = w, w + NW, ...
  constexpr int NS = 8 * MT / NW;  // chunks staged per wave
  static_assert(NS >= 1 && NS * NW == 8 * MT, "staging split");
  const uint16_t* wp = g.W + (size_t)(active ? nb : 0) * 2048 + (size_t)lane * 8;
  const size_t wstep = (size_t)nblk * 2048;  // next k-step of the same column block
  const uint16_t* sap[NS];
  int s_pl[NS], s_mt[NS], s_ch[NS];
#pragma unroll
  for (int j = 0; j < NS; ++j) {
    const int q = wave + NW * j;
    s_ch[j] = q & 3;
    s_mt[j] = (q >> 2) % MT;
    s_pl[j] = (q >> 2) / MT;
    sap[j] = (s_pl[j] ? g.A_lo : g.A) + (size_t)(s_mt[j] * 32 + r32) * g.lda + half * 32 + s_ch[j] * 8;
  }

  f32x16 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[mt][r] = 0.0f;
  u32x4 w[kRing][4], ra[kRing][NS];
  // step t of this workgroup's range, clamped to the last real step
  auto kstep = [&](int t) { return st0 + (t < n ? t : n - 1); };
  // steps past the range read 4 KB of the (cache-resident, finite) A plane
  // in place of a weight tile: they are multiplied by a zero tile
  const uint16_t* wpad = g.A + (size_t)lane * 8;
  auto issue = [&](int t, int slot) {
    const int st = kstep(t);
#pragma unroll
    for (int j = 0; j < NS; ++j) ra[slot][j] = *(const u32x4*)(sap[j] + st * 64);
    const uint16_t* src = t < n ? wp + (size_t)st * wstep : wpad;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[slot][i] = __builtin_nontemporal_load((const u32x4*)(src + i * 512));
  };
  auto stage = [&](int t, int slot, int buf) {
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < NS; ++j) sm.a[buf][s_pl[j]][s_mt[j]][s_ch[j]][lane] = t < n ? ra[slot][j] : z;
  };

  if (n > 0) {
#pragma unroll
    for (int t = 0; t < kRing - 1; ++t) issue(t, t);
    stage(0, 0, 0);
  }
  __syncthreads();
  for (int t0 = 0; t0 < npad; t0 += kRing) {
#pragma unroll
    for (int u = 0; u < kRing; ++u) {
      issue(t0 + u + kRing - 1, (u + kRing - 1) % kRing);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const u32x4 ah = sm.a[u & 1][0][mt][i][lane], al = sm.a[u & 1][1][mt][i][lane];
          acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ah), as_bf16x8(w[u][i]), acc[mt], 0, 0, 0);
          acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(al), as_bf16x8(w[u][i]), acc[mt], 0, 0, 0);
        }
      stage(t0 + u + 1, (u + 1) % kRing, (u + 1) & 1);
      __syncthreads();
    }
  }

  if (threadIdx.x < 32 * MT) {
    float ssum = 0.0f;
    if (has_ss) {
#pragma unroll
      for (int c = 0; c < kSsRegs; ++c) ssum += c < g.ss_n ? ssv[c] : 0.0f;
      for (int c = kSsRegs; c < g.ss_n; ++c) ssum += ssr[c];
    }
    sm.inv[threadIdx.x] = has_ss ? rsqrtf(ssum * g.inv_d + g.eps) : 1.0f;
  }
  __syncthreads();
  if (!active) return;
  // accumulator register r of lane l holds row 8(r/4) + 4(l/32) + r%4 of
  // its row tile, column l%32
  float* out = g.out + (size_t)sp * g.plane + (size_t)nb * 32 + r32;
  if ((MT & 1) == 0 && g.cfg_rows > 0) {
    // guided head: image b's text row 64b + m and unconditional row 64b +
    // 32 + m share lane and register; the guided row goes to row 32b + m
#pragma unroll
    for (int b = 0; b < MT / 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = 8 * (r / 4) + 4 * half + (r % 4);
        const float c = acc[2 * b][r] * sm.inv[64 * b + m], u = acc[2 * b + 1][r] * sm.inv[64 * b + 32 + m];
        if (m < g.cfg_rows) out[(size_t)(32 * b + m) * g.ldo] = u + g.cfg_w * (c - u);
      }
    return;
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = mt * 32 + 8 * (r / 4) + 4 * half + (r % 4);
      if (m < g.M) out[(size_t)m * g.ldo] = acc[mt][r] * sm.inv[m];
    }
}

// Split count along K. Splits that divide the K steps evenly are preferred
// (an uneven split leaves a tail of workgroups one step longer); among them
// the one whose workgroup count is nearest the target (by ratio), if within
// a factor of two, else ceil(0.8 target / groups).
int gemm_splits(int N, int K, int target_wgs, bool wide) {
  const int nw = wide ? kGWavesWide : kGWaves;
  const int groups = (N / 32 + nw - 1) / nw;
  const int T = K / 64;
  int smax = T / 2 > 0 ? T / 2 : 1;  // at least two k-steps per workgroup
  if (smax > kGemmMaxSplits) smax = kGemmMaxSplits;
  int best = 0;
  double best_r = 0.0;
  for (int S = 1; S <= smax; ++S) {
    if (T % S) continue;
    const double w = (double)groups * S;
    const double r = w > target_wgs ? w / target_wgs : target_wgs / w;
    if (best == 0 || r < best_r) {
      best = S;
      best_r = r;
    }
  }
  if (best > 0 && best_r <= 2.0) return best;
  // no even split near the target: stay below it (uneven splits add a tail)
  const int t2 = target_wgs * 4 / 5;
  int S = (t2 + groups - 1) / groups;
  if (S > smax) S = smax;
  if (S < 1) S = 1;
  return S;
}

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M < 1 || g.M > 128 || g.N % 32 || g.K % 64 || g.S < 1 || g.S > kGemmMaxSplits) return hipErrorInvalidValue;
  const int MT = (g.M + 31) / 32;
  if (g.cfg_rows < 0 || g.cfg_rows > 32 || (g.cfg_rows > 0 && (MT & 1))) return hipErrorInvalidValue;
  const int nw = g.wide ? kGWavesWide : kGWaves;
  const dim3 grid((unsigned)(((g.N / 32 + nw - 1) / nw) * g.S)), block((unsigned)(nw * kWave));
  // at one workgroup per compute unit or fewer nothing else hides a
  // workgroup's load latency: keep more weight tiles in flight
  const bool lone = grid.x <= 256;
  if (g.wide) {
    switch (MT) {
      case 1: hipLaunchKernelGGL((k_gemm<kRingDepth, 1, kGWavesWide>), grid, block, 0, s, g); break;
      case 2: hipLaunchKernelGGL((k_gemm<kRingDepth, 2, kGWavesWide>), grid, block, 0, s, g); break;
      case 3: hipLaunchKernelGGL((k_gemm<kRingDepth, 3, kGWavesWide>), grid, block, 0, s, g); break;
      default: hipLaunchKernelGGL((k_gemm<kRingDepth, 4, kGWavesWide>), grid, block, 0, s, g); break;
    }
  } else {
    switch (MT) {
      case 1:
        if (lone) hipLaunchKernelGGL((k_gemm<kRingDeep, 1, kGWaves>), grid, block, 0, s, g);
        else hipLaunchKernelGGL((k_gemm<kRingDepth, 1, kGWaves>), grid, block, 0, s, g);
        break;
      case 2: hipLaunchKernelGGL((k_gemm<kRingDepth, 2, kGWaves>), grid, block, 0, s, g); break;
      case 3: hipLaunchKernelGGL((k_gemm<kRingDepth, 3, kGWaves>), grid, block, 0, s, g); break;
      default: hipLaunchKernelGGL((k_gemm<kRingDepth, 4, kGWaves>), grid, block, 0, s, g); break;
    }
  }
  return hipGetLastError();
}

}  // namespace sjd
