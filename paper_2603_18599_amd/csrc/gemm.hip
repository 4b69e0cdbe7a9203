// Skinny bf16 GEMM for the window forward: C[M x N] = A[M x K] . W[N x K]^T
// with M <= 64 window slots, on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// The window forward is bound by streaming the weights from HBM (2 flop per
// weight byte per slot: 64 flop/B at M = 32, far below the MFMA ridge), so
// the kernel is laid out for the weight stream:
//  - weights are pre-tiled (see forward.h): a wave reads one 32-row x 64-k
//    tile per k-step as four contiguous 1 KB loads, prefetched two k-steps
//    ahead;
//  - the contraction index is permuted identically in A and W (any
//    permutation of k leaves the sum unchanged), so both operands load as
//    16-byte chunks straight into the MFMA register layout;
//  - a workgroup (4 waves) owns 32 output columns (64 for SwiGLU: the gate
//    and up rows of the same columns) and a K range split across its waves,
//    reduced in LDS. Long K is split across S workgroups that write
//    separate fp32 partial planes; the kernel that consumes the result sums
//    the planes in a fixed order (deterministic, and no device-scope fence,
//    which on this part would write back and invalidate the L2).
// Activations arrive as two bf16 planes (hi + lo, about 16 significant
// bits): the weights are exact bf16, so two MFMAs per tile recover an
// fp32-class product at no HBM cost (the MFMA units are otherwise idle).
// Epilogues: store fp32 (partial plane sp), SwiGLU -> hi / lo planes (S = 1).
#include "device.h"
#include "forward.h"

namespace sjd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGB = 256;
constexpr int kGWaves = kGB / kWave;

SJD_DEV bf16x8 as_bf16x8(const u32x4& u) { return __builtin_bit_cast(bf16x8, u); }

template <int MT, int NT>
struct GemmSmem {
  float red[kGWaves][MT][NT][16][kWave];
};

template <int MT, int MODE>
__global__ __launch_bounds__(kGB) void k_gemm(GemmArgs g) {
  constexpr int NT = (MODE == kGemmSwiGLU) ? 2 : 1;
  __shared__ GemmSmem<MT, NT> sm;
  const int nb = blockIdx.x, sp = blockIdx.y;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int r32 = lane & 31, half = lane >> 5;
  const int col0 = nb * 32;
  const int T = g.K / 64;

  // tile (nb, st) of each weight matrix; lane offset inside a tile
  const uint16_t* wp[NT];
  wp[0] = g.W0 + (size_t)nb * T * 2048 + (size_t)lane * 8;
  if constexpr (NT == 2) wp[1] = g.W1 + (size_t)nb * T * 2048 + (size_t)lane * 8;
  const uint16_t* ap[MT];
  const uint16_t* alp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    ap[mt] = g.A + (size_t)(mt * 32 + r32) * g.lda + half * 32;
    alp[mt] = g.A_lo + (size_t)(mt * 32 + r32) * g.lda + half * 32;
  }
  const int parts = g.S * kGWaves;
  const int part = sp * kGWaves + wave;
  const int st0 = (int)((long)T * part / parts);
  const int st1 = (int)((long)T * (part + 1) / parts);

  f32x16 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mt][t][r] = 0.0f;

  auto load_w = [&](int st, u32x4 (&w)[NT][4]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const uint16_t* tp = wp[t] + (size_t)st * 2048;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[t][i] = __builtin_nontemporal_load((const u32x4*)(tp + i * 512));
    }
  };
  auto load_a = [&](int st, u32x4 (&a)[MT][4], u32x4 (&al)[MT][4]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const u32x4* p = (const u32x4*)(ap[mt] + st * 64);
      const u32x4* pl = (const u32x4*)(alp[mt] + st * 64);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[mt][i] = p[i];
        al[mt][i] = pl[i];
      }
    }
  };
  // software pipeline: weights two k-steps ahead, activations one
  u32x4 w0[NT][4], w1[NT][4], a0[MT][4], al0[MT][4];
  if (st0 < st1) {
    load_w(st0, w0);
    load_a(st0, a0, al0);
  }
  if (st0 + 1 < st1) load_w(st0 + 1, w1);
  for (int st = st0; st < st1; ++st) {
    u32x4 w2[NT][4], a1[MT][4], al1[MT][4];
    if (st + 2 < st1) load_w(st + 2, w2);
    if (st + 1 < st1) load_a(st + 1, a1, al1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          acc[mt][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a0[mt][i]), as_bf16x8(w0[t][i]),
                                                               acc[mt][t], 0, 0, 0);
          acc[mt][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(al0[mt][i]), as_bf16x8(w0[t][i]),
                                                               acc[mt][t], 0, 0, 0);
        }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w0[t][i] = w1[t][i];
        w1[t][i] = w2[t][i];
      }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a0[mt][i] = a1[mt][i];
        al0[mt][i] = al1[mt][i];
      }
  }

  // ---- reduce the four waves in LDS
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) sm.red[wave][mt][t][r][lane] = acc[mt][t][r];
  __syncthreads();
  constexpr int E = MT * 16 * kWave;  // elements per tile per B-tile
  constexpr int PER = E / kGB;        // per thread
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = threadIdx.x + q * kGB;
    const int mt = e / (16 * kWave), r = (e / kWave) % 16, ln = e % kWave;
    float v[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < kGWaves; ++w) s += sm.red[w][mt][t][r][ln];
      v[t] = s;
    }
    const int m = mt * 32 + 8 * (r / 4) + 4 * (ln / 32) + (r % 4);
    const int n = col0 + (ln & 31);
    if (m >= g.M) continue;
    if constexpr (MODE == kGemmStore) {
      g.out[(size_t)sp * g.plane + (size_t)m * g.ldo + n] = v[0];
    } else {
      const float gt = v[0], up = v[1];
      const float h = gt / (1.0f + expf(-gt)) * up;
      split_bf16(h, g.outb[(size_t)m * g.ldo + n], g.outb_lo[(size_t)m * g.ldo + n]);
    }
  }
}

int gemm_splits(int N, int K, int target_wgs) {
  const int nblk = N / 32;
  const int T = K / 64;
  int S = (target_wgs + nblk - 1) / nblk;
  const int smax = T / (2 * kGWaves) > 0 ? T / (2 * kGWaves) : 1;  // at least two k-steps per wave
  if (S > smax) S = smax;
  if (S < 1) S = 1;
  return S;
}

hipError_t launch_gemm(const GemmArgs& g, int mode, hipStream_t s) {
  if (mode == kGemmSwiGLU && g.S != 1) return hipErrorInvalidValue;
  const dim3 grid(g.N / 32, g.S);
  const int MT = g.M > 32 ? 2 : 1;
  if (mode == kGemmStore) {
    if (MT == 1) hipLaunchKernelGGL((k_gemm<1, kGemmStore>), grid, dim3(kGB), 0, s, g);
    else hipLaunchKernelGGL((k_gemm<2, kGemmStore>), grid, dim3(kGB), 0, s, g);
  } else {
    if (MT == 1) hipLaunchKernelGGL((k_gemm<1, kGemmSwiGLU>), grid, dim3(kGB), 0, s, g);
    else hipLaunchKernelGGL((k_gemm<2, kGemmSwiGLU>), grid, dim3(kGB), 0, s, g);
  }
  return hipGetLastError();
}

}  // namespace sjd
