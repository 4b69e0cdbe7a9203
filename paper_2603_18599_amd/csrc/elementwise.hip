// Small kernels of the window forward: embedding gather, RMSNorm, rotary
// embedding with the key/value cache write, and weight conversion.
#include "device.h"
#include "forward.h"

namespace sjd {

// x[m][:] = E[tok[m]][:] (fp32 residual stream); d is a multiple of 64, so
// every 8-element chunk is whole. Token ids come from callers (prompts,
// drafts); an id outside [0, vocab) is read as token `fallback`, so no read
// leaves the embedding table.
__global__ __launch_bounds__(256) void k_embed(const uint16_t* E, const Window* win, int d, int vocab, int fallback,
                                               float* x) {
  const int m = blockIdx.x;
  int t = win->tok[m];
  t = (t >= 0 && t < vocab) ? t : fallback;
  const uint4* row = (const uint4*)(E + (size_t)t * d);
  float4* xr = (float4*)(x + (size_t)m * d);
  for (int c = threadIdx.x; c < d / 8; c += blockDim.x) {
    const uint4 u = row[c];
    xr[2 * c] = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                            __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
    xr[2 * c + 1] = make_float4(__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xFFFF0000u),
                                __uint_as_float(u.w << 16), __uint_as_float(u.w & 0xFFFF0000u));
  }
}

hipError_t launch_embed(const uint16_t* E, const Window* win, int M, int d, int vocab, int fallback, float* x,
                        hipStream_t s) {
  if (fallback < 0 || fallback >= vocab) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed, dim3(M), dim3(256), 0, s, E, win, d, vocab, fallback, x);
  return hipGetLastError();
}

// x += sum_s part[s] (split-K partial planes of the projection that feeds
// the residual, fixed order), y = x * g as hi / lo bf16 planes, ss[m][c] =
// sum of x^2 over the 256 elements of chunk c. grid (chunks, M), one wave.
// The planes were written moments ago by workgroups on every XCD, so each
// load is a far-memory round trip: all SMAX loads are issued at once
// (planes past S re-read the last plane and are not added).
template <int SMAX>
__global__ __launch_bounds__(64) void k_resid_norm(float* x, const float* part, int S, size_t plane,
                                                   const uint16_t* g, int d, uint16_t* y, uint16_t* y_lo, int ldy,
                                                   float* ss) {
  const int c = blockIdx.x, m = blockIdx.y, lane = threadIdx.x;
  const int i0 = c * 256 + lane * 4;
  float ssq = 0.0f;
  if (i0 < d) {  // d is a multiple of 64, so a lane's 4 elements are all in range
    float* xr = x + (size_t)m * d + i0;
    float4 v = *(const float4*)xr;
    if (S > 0) {
      const float* pr = part + (size_t)m * d + i0;
      float4 p[SMAX];
#pragma unroll
      for (int s = 0; s < SMAX; ++s) p[s] = *(const float4*)(pr + (size_t)(s < S ? s : S - 1) * plane);
#pragma unroll
      for (int s = 0; s < SMAX; ++s)
        if (s < S) {
          v.x += p[s].x;
          v.y += p[s].y;
          v.z += p[s].z;
          v.w += p[s].w;
        }
    }
    if (S > 0) *(float4*)xr = v;
    ssq = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    const ushort4 gg = *(const ushort4*)(g + i0);
    ushort4 h, l;
    split_bf16(v.x * bf16_to_f32(gg.x), h.x, l.x);
    split_bf16(v.y * bf16_to_f32(gg.y), h.y, l.y);
    split_bf16(v.z * bf16_to_f32(gg.z), h.z, l.z);
    split_bf16(v.w * bf16_to_f32(gg.w), h.w, l.w);
    *(ushort4*)(y + (size_t)m * ldy + i0) = h;
    *(ushort4*)(y_lo + (size_t)m * ldy + i0) = l;
  }
  ssq = wave_sum(ssq);
  if (lane == 0) ss[(size_t)m * gridDim.x + c] = ssq;
}

hipError_t launch_resid_norm(float* x, const float* part, int S, size_t plane, const uint16_t* g, int M, int d,
                             uint16_t* y, uint16_t* y_lo, int ldy, float* ss, hipStream_t s) {
  const dim3 grid(norm_chunks(d), M);
  if (S <= 4)
    hipLaunchKernelGGL(k_resid_norm<4>, grid, dim3(64), 0, s, x, part, S, plane, g, d, y, y_lo, ldy, ss);
  else if (S <= 8)
    hipLaunchKernelGGL(k_resid_norm<8>, grid, dim3(64), 0, s, x, part, S, plane, g, d, y, y_lo, ldy, ss);
  else if (S <= 16)
    hipLaunchKernelGGL(k_resid_norm<16>, grid, dim3(64), 0, s, x, part, S, plane, g, d, y, y_lo, ldy, ss);
  else if (S <= kGemmMaxSplits)
    hipLaunchKernelGGL(k_resid_norm<kGemmMaxSplits>, grid, dim3(64), 0, s, x, part, S, plane, g, d, y, y_lo, ldy,
                       ss);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// Rotate-half rotary embedding (pair i with i + hd/2 at angle pos * theta^(-2i/hd),
// table rope[pos][i] = (cos, sin)), then: q -> q planes, k and v -> cache
// position n + m (tiled layout), all as hi / lo bf16 planes. Two-stream
// windows: row m is slot m & 31 of stream m >> 5, cached at that stream's
// own position in its own cache; padding rows get a zero q and no cache write.
// grid (H + 2 * Hkv, M), block hd / 2. Head-major: workgroups are dealt to
// the XCDs round-robin by launch index, so (with H + 2 Hkv a multiple of 8)
// every row of one head runs on one XCD. A cache tile interleaves the rows
// of 8 positions in each 16-byte chunk, and its lines then fill in one L2
// instead of leaving as partial lines from eight (the row-major grid wrote
// 5.8 MB per launch for about 1.5 MB of data, and the step took 60 us longer).
template <int SMAX>
__global__ void k_rope_kv(const float* qkv, int S, size_t plane, const Window* win, const int32_t* n_dev, int n_host,
                          int H, int Hkv, int hd, const float2* rope, KvPlanes o, int cap, Streams sm) {
  const int m = blockIdx.y, hh = blockIdx.x, i = threadIdx.x;
  const int half = hd / 2;
  const bool two = sm.mode != kStreamsOne;
  const int z = two ? m >> 5 : 0;
  const int loc = two ? (m & 31) : m;
  if (two && loc >= sm.L) {
    if (hh < H) {
      const size_t off = (size_t)m * H * hd + (size_t)hh * hd;
      o.q[off + i] = o.q_lo[off + i] = o.q[off + i + half] = o.q_lo[off + i + half] = 0;
    }
    return;
  }
  const int n = stream_rows(sm, n_dev ? *n_dev : n_host, z);
  const int row = n + loc;
  if (z) {
    o.kc += z * o.sstride;
    o.kc_lo += z * o.sstride;
    o.vt += z * o.sstride;
    o.vt_lo += z * o.sstride;
  }
  const int ld = (H + 2 * Hkv) * hd;
  const float* src = qkv + (size_t)m * ld + (size_t)hh * hd;
  // all plane loads in flight at once (see k_resid_norm)
  float pa[SMAX], pb[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    const size_t so = (size_t)(s < S ? s : S - 1) * plane;
    pa[s] = src[so + i];
    pb[s] = src[so + i + half];
  }
  float a = 0.0f, b = 0.0f;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < S) {
      a += pa[s];
      b += pb[s];
    }
  if (hh < H + Hkv) {
    const float2 cs = rope[(size_t)win->pos[m] * half + i];
    const float o0 = a * cs.x - b * cs.y;
    const float o1 = a * cs.y + b * cs.x;
    if (hh < H) {
      const size_t off = (size_t)m * H * hd + (size_t)hh * hd;
      split_bf16(o0, o.q[off + i], o.q_lo[off + i]);
      split_bf16(o1, o.q[off + i + half], o.q_lo[off + i + half]);
    } else {
      const size_t base = (size_t)(hh - H) * cap * hd;
      const size_t k0 = base + kv_key_off(row, i, hd), k1 = base + kv_key_off(row, i + half, hd);
      split_bf16(o0, o.kc[k0], o.kc_lo[k0]);
      split_bf16(o1, o.kc[k1], o.kc_lo[k1]);
    }
  } else {
    const size_t base = (size_t)(hh - H - Hkv) * cap * hd;
    const size_t v0 = base + kv_val_off(row, i, hd), v1 = base + kv_val_off(row, i + half, hd);
    split_bf16(a, o.vt[v0], o.vt_lo[v0]);
    split_bf16(b, o.vt[v1], o.vt_lo[v1]);
  }
}

hipError_t launch_rope_kv(const float* qkv, int S, size_t plane, const Window* win, const int32_t* n_dev, int n_host,
                          int M, int H, int Hkv, int hd, const float2* rope, const KvPlanes& o, int cap,
                          const Streams& sm, hipStream_t s) {
  const dim3 grid(H + 2 * Hkv, M), block(hd / 2);
  if (S < 1) return hipErrorInvalidValue;
  if (S <= 4)
    hipLaunchKernelGGL(k_rope_kv<4>, grid, block, 0, s, qkv, S, plane, win, n_dev, n_host, H, Hkv, hd, rope, o, cap, sm);
  else if (S <= 8)
    hipLaunchKernelGGL(k_rope_kv<8>, grid, block, 0, s, qkv, S, plane, win, n_dev, n_host, H, Hkv, hd, rope, o, cap, sm);
  else if (S <= 16)
    hipLaunchKernelGGL(k_rope_kv<16>, grid, block, 0, s, qkv, S, plane, win, n_dev, n_host, H, Hkv, hd, rope, o, cap,
                       sm);
  else if (S <= kGemmMaxSplits)
    hipLaunchKernelGGL(k_rope_kv<kGemmMaxSplits>, grid, block, 0, s, qkv, S, plane, win, n_dev, n_host, H, Hkv, hd,
                       rope, o, cap, sm);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// h[m][n] = silu(g) * u with g, u the plane sums of columns n and F + n.
// grid (chunks of 256 columns, M), one wave, 4 columns per lane.
// (all plane loads in flight at once, see k_resid_norm)
template <int SMAX>
__global__ __launch_bounds__(64) void k_swiglu(const float* P, int S, size_t plane, int F, uint16_t* h,
                                               uint16_t* h_lo, int ldh) {
  const int m = blockIdx.y;
  const int n0 = blockIdx.x * 256 + threadIdx.x * 4;
  if (n0 >= F) return;  // F is a multiple of 64: a lane's 4 columns are all in range
  const float* pg = P + (size_t)m * 2 * F + n0;
  float4 pa[SMAX], pb[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    const size_t so = (size_t)(s < S ? s : S - 1) * plane;
    pa[s] = *(const float4*)(pg + so);
    pb[s] = *(const float4*)(pg + so + F);
  }
  float4 gs = make_float4(0.f, 0.f, 0.f, 0.f), us = gs;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < S) {
      gs.x += pa[s].x; gs.y += pa[s].y; gs.z += pa[s].z; gs.w += pa[s].w;
      us.x += pb[s].x; us.y += pb[s].y; us.z += pb[s].z; us.w += pb[s].w;
    }
  ushort4 hi, lo;
  split_bf16(gs.x / (1.0f + expf(-gs.x)) * us.x, hi.x, lo.x);
  split_bf16(gs.y / (1.0f + expf(-gs.y)) * us.y, hi.y, lo.y);
  split_bf16(gs.z / (1.0f + expf(-gs.z)) * us.z, hi.z, lo.z);
  split_bf16(gs.w / (1.0f + expf(-gs.w)) * us.w, hi.w, lo.w);
  *(ushort4*)(h + (size_t)m * ldh + n0) = hi;
  *(ushort4*)(h_lo + (size_t)m * ldh + n0) = lo;
}

hipError_t launch_swiglu(const float* P, int S, size_t plane, int M, int F, uint16_t* h, uint16_t* h_lo, int ldh,
                         hipStream_t s) {
  const dim3 grid((F + 255) / 256, M);
  if (S < 1) return hipErrorInvalidValue;
  if (S <= 4)
    hipLaunchKernelGGL(k_swiglu<4>, grid, dim3(64), 0, s, P, S, plane, F, h, h_lo, ldh);
  else if (S <= 8)
    hipLaunchKernelGGL(k_swiglu<8>, grid, dim3(64), 0, s, P, S, plane, F, h, h_lo, ldh);
  else if (S <= 16)
    hipLaunchKernelGGL(k_swiglu<16>, grid, dim3(64), 0, s, P, S, plane, F, h, h_lo, ldh);
  else if (S <= kGemmMaxSplits)
    hipLaunchKernelGGL(k_swiglu<kGemmMaxSplits>, grid, dim3(64), 0, s, P, S, plane, F, h, h_lo, ldh);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// one thread per 8-element chunk of the tiled layout
__global__ void k_tile_weights(const void* src, int is_f32, size_t row0, int N, int K, uint16_t* dst,
                               int nblk_total, int nb0) {
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
    uint16_t* d = dst + ((kb * nblk_total + nb0 + nb) * 256 + within) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) d[e] = v[e];
  }
}

hipError_t launch_tile_weights(const void* src, int is_f32, size_t row0, int N, int K, uint16_t* dst,
                               int nblk_total, int nb0, hipStream_t s) {
  size_t n = (size_t)N / 32 * (K / 64) * 256;
  size_t blocks = (n + 255) / 256;
  if (blocks > 65535 * 8) blocks = 65535 * 8;
  hipLaunchKernelGGL(k_tile_weights, dim3((unsigned)blocks), dim3(256), 0, s, src, is_f32, row0, N, K, dst,
                     nblk_total, nb0);
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
