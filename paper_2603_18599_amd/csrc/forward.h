// Internal interface of the window-forward kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sjd {

enum { kGemmStore = 0, kGemmSwiGLU = 2 };

// Weights are repacked at init into 32-row x 64-column tiles (4 KB, bf16):
// tile (nb, kb) of a [N][K] matrix starts at element (nb * (K/64) + kb) *
// 2048 and holds, for i = 0..3 and lane l = 0..63, the 8 elements of row
// nb*32 + l%32, columns kb*64 + (l/32)*32 + i*8 .. +8 at (i*64 + l) * 8. A wave
// then reads one tile as four contiguous 1 KB loads.
struct GemmArgs {
  const uint16_t* A;     // activations as two bf16 planes (A = hi + lo), rows padded to
  const uint16_t* A_lo;  // 32 * ceil(M/32), row stride lda
  int lda;
  int M;
  const uint16_t* W0;  // tiled weights [N][K]; SwiGLU: W0 = gate, W1 = up (same columns)
  const uint16_t* W1;
  int N, K;            // N multiple of 32, K multiple of 64
  int S;               // workgroups along K (SwiGLU: 1)
  float* out;          // store: fp32 partial plane sp at out + sp * plane, row stride ldo
  size_t plane;
  uint16_t* outb;      // SwiGLU output as hi / lo bf16 planes, row stride ldo
  uint16_t* outb_lo;
  int ldo;
};

int gemm_splits(int N, int K, int target_wgs);
hipError_t launch_gemm(const GemmArgs& g, int mode, hipStream_t s);

// Repacks rows [row0, row0 + N) of a row-major [*][K] bf16 (or fp32, then
// rounded to nearest even) matrix into the tile layout above.
hipError_t launch_tile_weights(const void* src, int is_f32, size_t row0, int N, int K, uint16_t* dst,
                               hipStream_t s);

// Window description in device memory (written by the window builder).
struct Window {
  int32_t tok[64];
  int32_t pos[64];
  uint64_t anc[64];
};

// Device-resident decoding state of one context.
struct DevState {
  int32_t n;        // cached rows
  int32_t pending;  // last committed token (slot 0)
  int32_t n_s, D_in, n_q, g0, q_off, pad;
  int32_t spine[64];
  int32_t sib[64];  // [D][K-1]
  int32_t meta[8];  // last step's outcome
  int32_t tok[64];  // last step's committed tokens
};

struct AttnArgs {
  // every tensor below is a pair of bf16 planes (value = hi + lo)
  const uint16_t* q;     // [Mpad][H * hd], rotated
  const uint16_t* q_lo;
  const uint16_t* kc;    // [Hkv][cap][hd] key cache of this layer
  const uint16_t* kc_lo;
  const uint16_t* vt;    // [Hkv][hd][cap] transposed value cache of this layer
  const uint16_t* vt_lo;
  const Window* win;
  const int32_t* n_dev;  // cached rows before the window (device scalar), or NULL -> n_host
  int n_host;
  int M, H, Hkv, cap;
  float scale;
  float* ws_o;           // [H][nsplit_max][32][hd] partial outputs
  float* ws_ml;          // [H][nsplit_max][32][2]  partial max (log2 domain) and sum
  int nsplit_max;
  uint16_t* out;         // [Mpad][ldo]
  uint16_t* out_lo;
  int ldo;
};
constexpr int kAttnChunk = 256;  // keys per workgroup
hipError_t launch_attention(const AttnArgs& a, int hd, hipStream_t s);

// elementwise kernels
hipError_t launch_embed(const uint16_t* E, const Window* win, int M, int d, float* x, hipStream_t s);
// x += sum of S fp32 partial planes (fixed order; S may be 0), then
// y = x / sqrt(mean(x^2) + eps) * g as hi / lo bf16 planes (row stride ldy)
hipError_t launch_rmsnorm(float* x, const float* part, int S, size_t plane, const uint16_t* g, int M, int d,
                          float eps, uint16_t* y, uint16_t* y_lo, int ldy, hipStream_t s);
// rotary embedding of q and k, key row and transposed value column into the caches
struct KvPlanes {
  uint16_t *q, *q_lo, *kc, *kc_lo, *vt, *vt_lo;
};
// qkv: S fp32 partial planes [S][plane] summed in order
hipError_t launch_rope_kv(const float* qkv, int S, size_t plane, const Window* win, const int32_t* n_dev, int n_host,
                          int M, int H, int Hkv, int hd, const float2* rope, const KvPlanes& o, int cap,
                          hipStream_t s);
hipError_t launch_f32_to_bf16(const float* src, uint16_t* dst, size_t n, hipStream_t s);

}  // namespace sjd
