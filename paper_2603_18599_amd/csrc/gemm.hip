// Skinny bf16 GEMM for the window forward: C[M x N] = A[M x K] . W[N x K]^T
// with M <= 32 window slots, on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// The window forward is bound by streaming the weights from HBM (2 flop per
// weight byte per slot: 64 flop/B at M = 32, far below the MFMA ridge), so
// the kernel is laid out for the weight stream:
//  - weights are pre-tiled (see forward.h): a wave reads one 32-row x 64-k
//    tile per k-step as four contiguous 1 KB loads, kDepth k-steps in flight;
//  - the activation tile of a k-step (32 rows x 64 k, hi and lo planes, 8 KB)
//    is staged once per workgroup into LDS (double buffered) and shared by
//    the four waves, each of which owns a different 32-column block. Loading
//    A per wave from L2 instead costs twice the weight bytes again and halves
//    the achieved weight bandwidth;
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
// RMSNorm, whose gain is already folded into A), then store fp32 to plane sp.
#include "device.h"
#include "forward.h"

namespace sjd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGB = 256;
constexpr int kGWaves = kGB / kWave;
constexpr int kDepth = 3;  // weight k-steps in flight per wave

SJD_DEV bf16x8 as_bf16x8(const u32x4& u) { return __builtin_bit_cast(bf16x8, u); }

struct GemmSmem {
  u32x4 a[2][2][4][kWave];  // [buffer][hi / lo][16-byte chunk][lane]: one A tile in MFMA operand order
  float inv[32];
};

__global__ __launch_bounds__(kGB) void k_gemm(GemmArgs g) {
  __shared__ GemmSmem sm;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int r32 = lane & 31, half = lane >> 5;
  const int T = g.K / 64, nblk = g.N / 32;
  const int nb = blockIdx.x * kGWaves + wave;  // this wave's 32-column block
  const bool active = nb < nblk;
  const int sp = blockIdx.y;
  const int st0 = (int)((long)T * sp / g.S), st1 = (int)((long)T * (sp + 1) / g.S);

  // fused RMSNorm: row scale from the chunk sums of squares (loads issued
  // ahead of the weight stream, consumed after it)
  float ssum = 0.0f;
  const bool has_ss = g.ss != nullptr && (int)threadIdx.x < g.M;
  if (has_ss)
    for (int c = 0; c < g.ss_n; ++c) ssum += g.ss[(size_t)threadIdx.x * g.ss_n + c];

  // element (row r32, k = kb*64 + half*32 + i*8 + e) of a tile sits in chunk
  // i of lane r32 + 32*half; wave w stages chunk w of every lane
  const uint16_t* wp = g.W + (size_t)(active ? nb : 0) * T * 2048 + (size_t)lane * 8;
  const size_t aofs = (size_t)r32 * g.lda + half * 32 + wave * 8;
  const uint16_t* sap = g.A + aofs;
  const uint16_t* salp = g.A_lo + aofs;

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  u32x4 w[kDepth][4];
  auto load_w = [&](int st, int j) {
    if (!active) return;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[j][i] = __builtin_nontemporal_load((const u32x4*)(wp + (size_t)st * 2048 + i * 512));
  };

  u32x4 ra, ral;
  if (st0 < st1) {
    ra = *(const u32x4*)(sap + st0 * 64);
    ral = *(const u32x4*)(salp + st0 * 64);
  }
#pragma unroll
  for (int p = 0; p < kDepth - 1; ++p)
    if (st0 + p < st1) load_w(st0 + p, p);
  if (st0 < st1) {
    sm.a[0][0][wave][lane] = ra;
    sm.a[0][1][wave][lane] = ral;
  }
  __syncthreads();
  for (int st = st0; st < st1; st += kDepth) {
#pragma unroll
    for (int j = 0; j < kDepth; ++j) {
      const int cur = st + j;
      if (cur < st1) {  // uniform over the workgroup
        const int buf = (cur - st0) & 1;
        if (cur + kDepth - 1 < st1) load_w(cur + kDepth - 1, (j + kDepth - 1) % kDepth);
        if (cur + 1 < st1) {
          ra = *(const u32x4*)(sap + (cur + 1) * 64);
          ral = *(const u32x4*)(salp + (cur + 1) * 64);
        }
        if (active) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const u32x4 ah = sm.a[buf][0][i][lane], al = sm.a[buf][1][i][lane];
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ah), as_bf16x8(w[j][i]), acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(al), as_bf16x8(w[j][i]), acc, 0, 0, 0);
          }
        }
        if (cur + 1 < st1) {
          sm.a[buf ^ 1][0][wave][lane] = ra;
          sm.a[buf ^ 1][1][wave][lane] = ral;
        }
        __syncthreads();
      }
    }
  }

  if (threadIdx.x < 32) sm.inv[threadIdx.x] = has_ss ? rsqrtf(ssum * g.inv_d + g.eps) : 1.0f;
  __syncthreads();
  if (!active) return;
  // accumulator register r of lane l holds row 8(r/4) + 4(l/32) + r%4, column l%32
  float* out = g.out + (size_t)sp * g.plane + (size_t)nb * 32 + r32;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int m = 8 * (r / 4) + 4 * half + (r % 4);
    if (m < g.M) out[(size_t)m * g.ldo] = acc[r] * sm.inv[m];
  }
}

// Split count along K. Splits that divide the K steps evenly are preferred
// (an uneven split leaves a tail of workgroups one step longer); among them
// the one whose workgroup count is nearest the target (by ratio), if within
// a factor of two, else ceil(target / groups).
int gemm_splits(int N, int K, int target_wgs) {
  const int groups = (N / 32 + kGWaves - 1) / kGWaves;
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
  int S = (target_wgs + groups - 1) / groups;
  if (S > smax) S = smax;
  if (S < 1) S = 1;
  return S;
}

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M < 1 || g.M > 32 || g.N % 32 || g.K % 64 || g.S < 1 || g.S > kGemmMaxSplits) return hipErrorInvalidValue;
  const dim3 grid((g.N / 32 + kGWaves - 1) / kGWaves, g.S);
  hipLaunchKernelGGL(k_gemm, grid, dim3(kGB), 0, s, g);
  return hipGetLastError();
}

}  // namespace sjd
