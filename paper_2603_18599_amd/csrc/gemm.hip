// Skinny bf16 GEMM for the window forward: C[M x N] = A[M x K] . W[N x K]^T
// with M <= 64 window slots, on gfx950 MFMA (v_mfma_f32_32x32x16_bf16).
//
// The window forward is bound by streaming the weights from HBM (2 flop per
// weight byte per slot: 64 flop/B at M = 32, far below the MFMA ridge), so
// the kernel is laid out for the weight stream:
//  - each lane reads 64 contiguous bytes of one weight row per k-step; the
//    two lane halves cover 128 contiguous bytes, so a wave reads 32 rows x
//    128 B. The contraction index is permuted identically in A and W (any
//    permutation of k leaves the sum unchanged), which lets both operands be
//    loaded as 16-byte chunks straight into the MFMA register layout;
//  - a workgroup (4 waves) owns 32 output columns (64 for SwiGLU: the gate
//    and up rows of the same columns) and a K range split across its waves,
//    reduced in LDS; long K is further split across S workgroups whose
//    partials are summed in a fixed order by the last one to arrive
//    (deterministic, no float atomics);
//  - the next k-step's loads are issued before the current step's MFMAs.
// Activations arrive as two bf16 planes (hi + lo, about 16 significant
// bits): the weights are exact bf16, so two MFMAs per tile recover an
// fp32-class product at no HBM cost (the MFMA units are otherwise idle).
// Epilogues: store fp32, add into fp32 (residual), SwiGLU -> hi / lo planes.
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
  int last;
};

template <int MT, int MODE>
__global__ __launch_bounds__(kGB) void k_gemm(GemmArgs g) {
  constexpr int NT = (MODE == kGemmSwiGLU) ? 2 : 1;
  __shared__ GemmSmem<MT, NT> sm;
  const int nb = blockIdx.x, sp = blockIdx.y;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int r32 = lane & 31, half = lane >> 5;
  const int col0 = nb * 32;
  const int K = g.K;

  const uint16_t* wp[NT];
  if constexpr (MODE == kGemmSwiGLU) {
    wp[0] = g.W0 + (size_t)(col0 + r32) * K;
    wp[1] = g.W1 + (size_t)(col0 + r32) * K;
  } else {
    const int r = col0 + r32;
    wp[0] = r < g.n0 ? g.W0 + (size_t)r * K
                     : (r < g.n1 ? g.W1 + (size_t)(r - g.n0) * K : g.W2 + (size_t)(r - g.n1) * K);
  }
  const uint16_t* ap[MT];
  const uint16_t* alp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    ap[mt] = g.A + (size_t)(mt * 32 + r32) * K;
    alp[mt] = g.A_lo + (size_t)(mt * 32 + r32) * K;
  }

  const int T = K / 64;
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

  u32x4 wb[NT][4], ab[MT][4], alb[MT][4];
  auto load = [&](int st, u32x4 (&w)[NT][4], u32x4 (&a)[MT][4], u32x4 (&al)[MT][4]) {
    const int koff = st * 64 + half * 32;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const u32x4* p = (const u32x4*)(wp[t] + koff);
#pragma unroll
      for (int i = 0; i < 4; ++i) w[t][i] = __builtin_nontemporal_load(p + i);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const u32x4* p = (const u32x4*)(ap[mt] + koff);
      const u32x4* pl = (const u32x4*)(alp[mt] + koff);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[mt][i] = p[i];
        al[mt][i] = pl[i];
      }
    }
  };
  if (st0 < st1) load(st0, wb, ab, alb);
  for (int st = st0; st < st1; ++st) {
    u32x4 wn[NT][4], an[MT][4], aln[MT][4];
    if (st + 1 < st1) load(st + 1, wn, an, aln);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          acc[mt][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ab[mt][i]), as_bf16x8(wb[t][i]),
                                                               acc[mt][t], 0, 0, 0);
          acc[mt][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(alb[mt][i]), as_bf16x8(wb[t][i]),
                                                               acc[mt][t], 0, 0, 0);
        }
    if (st + 1 < st1) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) wb[t][i] = wn[t][i];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ab[mt][i] = an[mt][i];
          alb[mt][i] = aln[mt][i];
        }
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
  float v[PER][NT];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = threadIdx.x + q * kGB;
    const int mt = e / (16 * kWave), r = (e / kWave) % 16, ln = e % kWave;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < kGWaves; ++w) s += sm.red[w][mt][t][r][ln];
      v[q][t] = s;
    }
  }

  // ---- split-K across workgroups: the last arriver sums all partials in
  // split order
  if (g.S > 1) {
    float* part_base = g.ws + (size_t)nb * g.S * NT * E;
#pragma unroll
    for (int q = 0; q < PER; ++q)
#pragma unroll
      for (int t = 0; t < NT; ++t) part_base[((size_t)sp * NT + t) * E + threadIdx.x + q * kGB] = v[q][t];
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
      const int old = atomicAdd(g.cnt + nb, 1);
      sm.last = (old == g.S - 1);
    }
    __syncthreads();
    if (!sm.last) return;
    __threadfence();
#pragma unroll
    for (int q = 0; q < PER; ++q)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        float s = 0.0f;
        for (int k = 0; k < g.S; ++k)
          s += __builtin_nontemporal_load(part_base + ((size_t)k * NT + t) * E + threadIdx.x + q * kGB);
        v[q][t] = s;
      }
    if (threadIdx.x == 0) g.cnt[nb] = 0;
  }

  // ---- epilogue
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int e = threadIdx.x + q * kGB;
    const int mt = e / (16 * kWave), r = (e / kWave) % 16, ln = e % kWave;
    const int m = mt * 32 + 8 * (r / 4) + 4 * (ln / 32) + (r % 4);
    const int n = col0 + (ln & 31);
    if (m >= g.M) continue;
    if constexpr (MODE == kGemmStore) {
      g.out[(size_t)m * g.ldo + n] = v[q][0];
    } else if constexpr (MODE == kGemmAdd) {
      g.out[(size_t)m * g.ldo + n] += v[q][0];
    } else {
      const float gt = v[q][0], up = v[q][1];
      const float h = gt / (1.0f + expf(-gt)) * up;
      split_bf16(h, g.outb[(size_t)m * g.ldo + n], g.outb_lo[(size_t)m * g.ldo + n]);
    }
  }
}

size_t gemm_ws_floats(int N, int S, int M, int mode) {
  const int MT = M > 32 ? 2 : 1;
  const int NT = mode == kGemmSwiGLU ? 2 : 1;
  return S > 1 ? (size_t)(N / 32) * S * NT * MT * 16 * kWave : 0;
}

int gemm_splits(int N, int K, int target_wgs) {
  const int nblk = N / 32;
  const int T = K / 64;
  int S = (target_wgs + nblk - 1) / nblk;
  const int smax = T / kGWaves > 0 ? T / kGWaves : 1;  // at least one k-step per wave
  if (S > smax) S = smax;
  if (S < 1) S = 1;
  return S;
}

hipError_t launch_gemm(const GemmArgs& g, int mode, hipStream_t s) {
  const dim3 grid(g.N / 32, g.S);
  const int MT = g.M > 32 ? 2 : 1;
  if (mode == kGemmStore) {
    if (MT == 1) hipLaunchKernelGGL((k_gemm<1, kGemmStore>), grid, dim3(kGB), 0, s, g);
    else hipLaunchKernelGGL((k_gemm<2, kGemmStore>), grid, dim3(kGB), 0, s, g);
  } else if (mode == kGemmAdd) {
    if (MT == 1) hipLaunchKernelGGL((k_gemm<1, kGemmAdd>), grid, dim3(kGB), 0, s, g);
    else hipLaunchKernelGGL((k_gemm<2, kGemmAdd>), grid, dim3(kGB), 0, s, g);
  } else {
    if (MT == 1) hipLaunchKernelGGL((k_gemm<1, kGemmSwiGLU>), grid, dim3(kGB), 0, s, g);
    else hipLaunchKernelGGL((k_gemm<2, kGemmSwiGLU>), grid, dim3(kGB), 0, s, g);
  }
  return hipGetLastError();
}

}  // namespace sjd
