// Internal interface of the window-forward kernels (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sjd {

constexpr int kGemmMaxSplits = 32;

// Weights are repacked at init into 32-row x 64-column tiles (4 KB, bf16):
// tile (nb, kb) of a [N][K] matrix starts at element (kb * (N/32) + nb) *
// 2048 and holds, for i = 0..3 and lane l = 0..63, the 8 elements of row
// nb*32 + l%32, columns kb*64 + (l/32)*32 + i*8 .. +8 at (i*64 + l) * 8. A wave
// then reads one tile as four contiguous 1 KB loads, and the tiles that the
// column blocks read at the same k-step are adjacent (one contiguous stripe
// per k-step instead of tiles a whole row block apart, which measurably
// streams faster). Matrices that share an input (q, k, v; gate, up) are
// tiled as row blocks of one [N][K].
struct GemmArgs {
  const uint16_t* A;     // activations as two bf16 planes (A = hi + lo), 32 rows
  const uint16_t* A_lo;  // per started 32 (rows >= M finite), row stride lda
  int lda;
  int M;               // 1..128
  const uint16_t* W;   // tiled weights [N][K]
  int N, K;            // N multiple of 32, K multiple of 64
  int S;               // workgroups along K = fp32 partial planes (1..kGemmMaxSplits)
  float* out;          // plane sp at out + sp * plane, row stride ldo
  size_t plane;
  int ldo;
  // optional RMS scale of row m (fused RMSNorm): rsqrt(sum_c ss[m * ss_n + c] *
  // inv_d + eps) multiplies the row of the product before the store
  const float* ss;
  int ss_n;
  float inv_d, eps;
  // guided head (M > 32 only): for each image b (product rows [64 b, 64 b +
  // 64)), output row 32 b + m (m < cfg_rows) is u + cfg_w (c - u) with c =
  // product row 64 b + m, u = product row 64 b + 32 + m
  int cfg_rows;
  float cfg_w;
  // 8 column blocks per workgroup (else 4): half the activation loads per
  // weight byte; the grid is N / 256 column groups x S
  int wide;
};

// splits for about target_wgs workgroups of 4 (or, wide, 8) column blocks
int gemm_splits(int N, int K, int target_wgs, bool wide);
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s);

// Repacks rows [row0, row0 + N) of a row-major [*][K] bf16 (or fp32, then
// rounded to nearest even) matrix into the tile layout above, as row blocks
// [nb0, nb0 + N/32) of a tiled matrix of nblk_total row blocks at dst.
hipError_t launch_tile_weights(const void* src, int is_f32, size_t row0, int N, int K, uint16_t* dst,
                               int nblk_total, int nb0, hipStream_t s);

// Window description in device memory (written by the window builder).
// Row a's ancestors: bit i = row base + i of its own stream (base 0 for
// one stream, 32 z for stream z), a row itself included.
constexpr int kWinRows = 128;
struct Window {
  int32_t tok[kWinRows];
  int32_t pos[kWinRows];
  uint64_t anc[kWinRows];
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
  int32_t pending_u;  // guided contexts: pending token of the unconditional stream
  int32_t delta_u;    // guided contexts: unconditional-stream position minus text-stream position
  int32_t pad2[2];
};

// A window forward runs one stream (rows [0, M)) or nz <= 4 streams of L <=
// 32 rows each: stream z at rows [32 z, 32 z + L), the other rows padding
// (never cached, never read). Each stream has its own key/value cache
// (stream z's at the stream-0 cache + z * sstride) and its own positions:
//  - batched: stream z is image z, with its own decoder state;
//  - guided (classifier-free guidance): streams come in pairs per image,
//    2b the text stream and 2b + 1 the unconditional stream, which is fed
//    the same window tokens (its own first pending token) at positions
//    shifted by the image's delta_u.
enum { kStreamsOne = 0, kStreamsMulti = 1 };
constexpr int kMaxStreams = 4;
struct Streams {
  int mode;            // kStreams*
  int L;               // window rows per stream (multi)
  int nz;              // streams (multi)
  int guided;          // multi: (text, unconditional) stream pairs
  const DevState* st;  // multi: decoder state of image 0 (image b at st + b)
};
__device__ inline int stream_image(const Streams& sm, int z) { return sm.guided ? z >> 1 : z; }
__device__ inline bool stream_uncond(const Streams& sm, int z) { return sm.guided && (z & 1); }
// cached rows before the window of stream z (one stream: n0)
__device__ inline int stream_rows(const Streams& sm, int n0, int z) {
  if (sm.mode == kStreamsOne) return n0;
  const DevState& d = sm.st[stream_image(sm, z)];
  return d.n + (stream_uncond(sm, z) ? d.delta_u : 0);
}

// Key / value cache layout. Per layer and kv head, positions are grouped in
// tiles of 32 (32 * hd elements each) stored in the register order of the
// attention MFMAs, so that every load of a tile is a contiguous 1 KB per
// wave: key (position p, dim j) is element (t * 64 + lane) * 8 + e of tile
// p / 32, with lane = swap23(p % 32) + 32 * (j / (hd / 2)), t = (j % (hd / 2)) / 8,
// e = j % 8 (swap23 exchanges bits 2 and 3: the key-row order of the score
// MFMA); value (p, j) is element ((j / 32) * 2 + i / 16) * 512 + lane * 8 + i % 8
// with i = p % 32, lane = j % 32 + 32 * ((i / 8) % 2) (the transposed-value
// operand of the output MFMA).
__host__ __device__ inline int swap23(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }
__host__ __device__ inline size_t kv_key_off(int p, int j, int hd) {
  const int i = p & 31, h2 = hd / 2;
  const int lane = swap23(i) + 32 * (j / h2), t = (j % h2) >> 3;
  return (size_t)(p >> 5) * 32 * hd + (size_t)(t * 64 + lane) * 8 + (j & 7);
}
__host__ __device__ inline size_t kv_val_off(int p, int j, int hd) {
  const int i = p & 31;
  const int lane = (j & 31) + 32 * ((i >> 3) & 1);
  return (size_t)(p >> 5) * 32 * hd + (size_t)(((j >> 5) * 2 + (i >> 4)) * 64 + lane) * 8 + (i & 7);
}

struct AttnArgs {
  // every tensor below is a pair of bf16 planes (value = hi + lo)
  const uint16_t* q;     // [Mpad][H * hd], rotated
  const uint16_t* q_lo;
  const uint16_t* kc;    // [Hkv][cap * hd] key cache of this layer (tiled, see above)
  const uint16_t* kc_lo;
  const uint16_t* vt;    // [Hkv][cap * hd] value cache of this layer (tiled)
  const uint16_t* vt_lo;
  size_t sstride;        // multi-stream windows: stream z's caches are these + z * sstride
  Streams st;
  const Window* win;
  const int32_t* n_dev;  // cached rows before the window (device scalar), or NULL -> n_host
  int n_host;
  int M, H, Hkv, cap;
  float scale;
  float* ws_o;           // [H][nsplit_max][128][hd] partial outputs (per query slot)
  float* ws_ml;          // [H][nsplit_max][128][2]  partial max (log2 domain) and sum
  int nsplit_max;
  uint16_t* out;         // [Mpad][ldo]
  uint16_t* out_lo;
  int ldo;
  int qparts;            // workgroups per key / value head, each taking H / Hkv / qparts query heads
};
constexpr int kAttnChunk = 128;  // keys per workgroup (4 waves x 32)
hipError_t launch_attention(const AttnArgs& a, int hd, hipStream_t s);

// elementwise kernels
// ids outside [0, vocab) are read as token fallback (in [0, vocab))
hipError_t launch_embed(const uint16_t* E, const Window* win, int M, int d, int vocab, int fallback, float* x,
                        hipStream_t s);
// RMSNorm split in two: x += sum of S fp32 partial planes (fixed order; S
// may be 0), y = x * g as hi / lo bf16 planes (row stride ldy) and the
// sums of squares of x over 256-element chunks, ss[m][c] (c < norm_chunks(d));
// the GEMM that consumes y applies the row scale 1 / sqrt(mean(x^2) + eps).
inline int norm_chunks(int d) { return (d + 255) / 256; }
hipError_t launch_resid_norm(float* x, const float* part, int S, size_t plane, const uint16_t* g, int M, int d,
                             uint16_t* y, uint16_t* y_lo, int ldy, float* ss, hipStream_t s);
// rotary embedding of q and k, key row and transposed value column into the caches
struct KvPlanes {
  uint16_t *q, *q_lo, *kc, *kc_lo, *vt, *vt_lo;
  size_t sstride;  // multi-stream windows: stream z's caches are kc.. + z * sstride
};
// qkv: S fp32 partial planes [S][plane] summed in order
hipError_t launch_rope_kv(const float* qkv, int S, size_t plane, const Window* win, const int32_t* n_dev, int n_host,
                          int M, int H, int Hkv, int hd, const float2* rope, const KvPlanes& o, int cap,
                          const Streams& st, hipStream_t s);
// h = silu(gate) * up as hi / lo bf16 planes (row stride ldh), gate = sum of
// the S fp32 partial planes at columns [0, F), up = at columns [F, 2F)
// (row stride 2F)
hipError_t launch_swiglu(const float* P, int S, size_t plane, int M, int F, uint16_t* h, uint16_t* h_lo, int ldh,
                         hipStream_t s);
hipError_t launch_f32_to_bf16(const float* src, uint16_t* dst, size_t n, hipStream_t s);

}  // namespace sjd
