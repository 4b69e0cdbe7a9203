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

// y = bf16(x / sqrt(mean(x^2) + eps) * g), one workgroup per row
__global__ __launch_bounds__(256) void k_rmsnorm(const float* x, const uint16_t* g, int d, float eps, uint16_t* y) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* xr = x + (size_t)m * d;
  float ss = 0.0f;
  for (int i = threadIdx.x; i < d; i += 256) ss += xr[i] * xr[i];
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = rsqrtf(tot / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256) y[(size_t)m * d + i] = f32_to_bf16(xr[i] * inv * bf16_to_f32(g[i]));
}

hipError_t launch_rmsnorm(const float* x, const uint16_t* g, int M, int d, float eps, uint16_t* y, hipStream_t s) {
  hipLaunchKernelGGL(k_rmsnorm, dim3(M), dim3(256), 0, s, x, g, d, eps, y);
  return hipGetLastError();
}

// Rotate-half rotary embedding (pair i with i + hd/2 at angle pos * theta^(-2i/hd),
// table rope[pos][i] = (cos, sin)), then: q -> q buffer (bf16), k -> key cache
// row n + m, v -> column n + m of the transposed value cache.
// grid (M, H + 2 * Hkv), block hd / 2
__global__ void k_rope_kv(const float* qkv, const Window* win, const int32_t* n_dev, int n_host, int H, int Hkv,
                          int hd, const float2* rope, uint16_t* q, uint16_t* kc, uint16_t* vt, int cap) {
  const int m = blockIdx.x, hh = blockIdx.y, i = threadIdx.x;
  const int half = hd / 2;
  const int n = n_dev ? *n_dev : n_host;
  const int row = n + m;
  const int ld = (H + 2 * Hkv) * hd;
  const float* src = qkv + (size_t)m * ld + (size_t)hh * hd;
  if (hh < H + Hkv) {
    const float2 cs = rope[(size_t)win->pos[m] * half + i];
    const float a = src[i], b = src[i + half];
    const float o0 = a * cs.x - b * cs.y;
    const float o1 = a * cs.y + b * cs.x;
    if (hh < H) {
      uint16_t* dst = q + (size_t)m * H * hd + (size_t)hh * hd;
      dst[i] = f32_to_bf16(o0);
      dst[i + half] = f32_to_bf16(o1);
    } else {
      const int kh = hh - H;
      uint16_t* dst = kc + ((size_t)kh * cap + row) * hd;
      dst[i] = f32_to_bf16(o0);
      dst[i + half] = f32_to_bf16(o1);
    }
  } else {
    const int vh = hh - H - Hkv;
    uint16_t* dst = vt + (size_t)vh * hd * cap;
    dst[(size_t)i * cap + row] = f32_to_bf16(src[i]);
    dst[(size_t)(i + half) * cap + row] = f32_to_bf16(src[i + half]);
  }
}

hipError_t launch_rope_kv(const float* qkv, const Window* win, const int32_t* n_dev, int n_host, int M, int H,
                          int Hkv, int hd, const float2* rope, uint16_t* q, uint16_t* kc, uint16_t* vt, int cap,
                          hipStream_t s) {
  hipLaunchKernelGGL(k_rope_kv, dim3(M, H + 2 * Hkv), dim3(hd / 2), 0, s, qkv, win, n_dev, n_host, H, Hkv, hd, rope,
                     q, kc, vt, cap);
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
