// Small kernels of the window forward: embedding gather, RMSNorm, rotary
// embedding with the key/value cache write, and weight conversion.
#include "device.h"
#include "forward.h"

namespace sjd {

// x[m][:] = E[tok[m]][:] (fp32 residual stream)
__global__ __launch_bounds__(256) void k_embed(const uint16_t* E, const Window* win, int d, float* x) {
  const int m = blockIdx.x;
  const int t = win->tok[m];
  const uint16_t* row = E + (size_t)t * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)m * d + i] = bf16_to_f32(row[i]);
}

hipError_t launch_embed(const uint16_t* E, const Window* win, int M, int d, float* x, hipStream_t s) {
  hipLaunchKernelGGL(k_embed, dim3(M), dim3(256), 0, s, E, win, d, x);
  return hipGetLastError();
}

// x += sum_s part[s] (split-K partial planes of the projection that feeds
// the residual, fixed order), then y = x / sqrt(mean(x^2) + eps) * g as hi /
// lo bf16 planes; one workgroup per row
__global__ __launch_bounds__(256) void k_rmsnorm(float* x, const float* part, int S, size_t plane,
                                                 const uint16_t* g, int d, float eps, uint16_t* y, uint16_t* y_lo,
                                                 int ldy) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  float* xr = x + (size_t)m * d;
  float ss = 0.0f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = xr[i];
    for (int s = 0; s < S; ++s) v += part[(size_t)s * plane + (size_t)m * d + i];
    if (S > 0) xr[i] = v;
    ss += v * v;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = rsqrtf(tot / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256)
    split_bf16(xr[i] * inv * bf16_to_f32(g[i]), y[(size_t)m * ldy + i], y_lo[(size_t)m * ldy + i]);
}

hipError_t launch_rmsnorm(float* x, const float* part, int S, size_t plane, const uint16_t* g, int M, int d,
                          float eps, uint16_t* y, uint16_t* y_lo, int ldy, hipStream_t s) {
  hipLaunchKernelGGL(k_rmsnorm, dim3(M), dim3(256), 0, s, x, part, S, plane, g, d, eps, y, y_lo, ldy);
  return hipGetLastError();
}

// Rotate-half rotary embedding (pair i with i + hd/2 at angle pos * theta^(-2i/hd),
// table rope[pos][i] = (cos, sin)), then: q -> q planes, k -> key cache row
// n + m, v -> column n + m of the transposed value cache, all as hi / lo bf16
// planes. grid (M, H + 2 * Hkv), block hd / 2
__global__ void k_rope_kv(const float* qkv, int S, size_t plane, const Window* win, const int32_t* n_dev, int n_host,
                          int H, int Hkv, int hd, const float2* rope, KvPlanes o, int cap) {
  const int m = blockIdx.x, hh = blockIdx.y, i = threadIdx.x;
  const int half = hd / 2;
  const int n = n_dev ? *n_dev : n_host;
  const int row = n + m;
  const int ld = (H + 2 * Hkv) * hd;
  const float* src = qkv + (size_t)m * ld + (size_t)hh * hd;
  float a = 0.0f, b = 0.0f;
  for (int s = 0; s < S; ++s) {
    a += src[(size_t)s * plane + i];
    b += src[(size_t)s * plane + i + half];
  }
  if (hh < H + Hkv) {
    const float2 cs = rope[(size_t)win->pos[m] * half + i];
    const float o0 = a * cs.x - b * cs.y;
    const float o1 = a * cs.y + b * cs.x;
    size_t off;
    uint16_t *dh, *dl;
    if (hh < H) {
      off = (size_t)m * H * hd + (size_t)hh * hd;
      dh = o.q; dl = o.q_lo;
    } else {
      off = ((size_t)(hh - H) * cap + row) * hd;
      dh = o.kc; dl = o.kc_lo;
    }
    split_bf16(o0, dh[off + i], dl[off + i]);
    split_bf16(o1, dh[off + i + half], dl[off + i + half]);
  } else {
    const size_t base = (size_t)(hh - H - Hkv) * hd * cap + row;
    split_bf16(a, o.vt[base + (size_t)i * cap], o.vt_lo[base + (size_t)i * cap]);
    split_bf16(b, o.vt[base + (size_t)(i + half) * cap], o.vt_lo[base + (size_t)(i + half) * cap]);
  }
}

hipError_t launch_rope_kv(const float* qkv, int S, size_t plane, const Window* win, const int32_t* n_dev, int n_host,
                          int M, int H, int Hkv, int hd, const float2* rope, const KvPlanes& o, int cap,
                          hipStream_t s) {
  hipLaunchKernelGGL(k_rope_kv, dim3(M, H + 2 * Hkv), dim3(hd / 2), 0, s, qkv, S, plane, win, n_dev, n_host, H, Hkv,
                     hd, rope, o, cap);
  return hipGetLastError();
}

// one thread per 8-element chunk of the tiled layout
__global__ void k_tile_weights(const void* src, int is_f32, size_t row0, int N, int K, uint16_t* dst) {
  const size_t T = (size_t)K / 64;
  const size_t nchunks = (size_t)N / 32 * T * 256;
  for (size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x; q < nchunks; q += (size_t)gridDim.x * blockDim.x) {
    const size_t tile = q / 256, within = q % 256;
    const int i = (int)(within / 64), l = (int)(within % 64);
    const size_t nb = tile / T, kb = tile % T;
    const size_t row = row0 + nb * 32 + (size_t)(l % 32);
    const size_t col = kb * 64 + (size_t)(l / 32) * 32 + (size_t)i * 8;
    uint16_t v[8];
    if (is_f32) {
      const float* p = (const float*)src + row * (size_t)K + col;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = f32_to_bf16(p[e]);
    } else {
      const uint16_t* p = (const uint16_t*)src + row * (size_t)K + col;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = p[e];
    }
    uint16_t* d = dst + q * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) d[e] = v[e];
  }
}

hipError_t launch_tile_weights(const void* src, int is_f32, size_t row0, int N, int K, uint16_t* dst,
                               hipStream_t s) {
  size_t n = (size_t)N / 32 * (K / 64) * 256;
  size_t blocks = (n + 255) / 256;
  if (blocks > 65535 * 8) blocks = 65535 * 8;
  hipLaunchKernelGGL(k_tile_weights, dim3((unsigned)blocks), dim3(256), 0, s, src, is_f32, row0, N, K, dst);
  return hipGetLastError();
}

__global__ void k_f32_to_bf16(const float* src, uint16_t* dst, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = f32_to_bf16(src[i]);
}

hipError_t launch_f32_to_bf16(const float* src, uint16_t* dst, size_t n, hipStream_t s) {
  size_t blocks = (n + 255) / 256;
  if (blocks > 65535 * 4) blocks = 65535 * 4;
  hipLaunchKernelGGL(k_f32_to_bf16, dim3((unsigned)blocks), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

}  // namespace sjd
