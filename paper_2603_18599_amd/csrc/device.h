// Device-side helpers shared by the HIP kernels of libsjd: Philox4x32-10,
// bf16 conversion, wave and block reductions. gfx950 (CDNA4), wave64.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define SJD_DEV __device__ __forceinline__

namespace sjd {

constexpr int kWave = 64;

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds, each
// multiplying counter words 0 and 2 by the two round constants and mixing the
// high halves with the other words and the key; the key advances by the Weyl
// constants between rounds.
SJD_DEV uint4 philox(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}

// Stream tags (counter word 2 bits 24..31).
enum : uint32_t { kTagAcc = 1, kTagRes = 2, kTagFresh = 3, kTagBonus = 4, kTagPd = 5, kTagInit = 6 };

struct Stream {
  uint32_t k0, k1, trial, w2, step;
  SJD_DEV Stream(uint64_t seed, uint32_t tag, uint32_t stage, uint32_t row, uint32_t trial_, uint32_t step_)
      : k0((uint32_t)seed), k1((uint32_t)(seed >> 32)), trial(trial_),
        w2((tag << 24) | ((stage & 0xFFu) << 16) | (row & 0xFFFFu)), step(step_) {}
  // the four words of elements 4*blk .. 4*blk+3
  SJD_DEV uint4 block(uint32_t blk) const { return philox(make_uint4(blk, trial, w2, step), k0, k1); }
  SJD_DEV uint32_t word(uint32_t x) const {
    uint4 b = block(x >> 2);
    uint32_t s = x & 3u;
    return s == 0 ? b.x : s == 1 ? b.y : s == 2 ? b.z : b.w;
  }
};

SJD_DEV float u01(uint32_t w) { return (float)(w >> 8) * 0x1p-24f; }
// Exp(1) variate; 1 - u is exact because u is a multiple of 2^-24.
SJD_DEV float exp1(uint32_t w) { return -logf(1.0f - u01(w)); }

// Order-preserving map of a float to uint32 (larger float -> larger key).
SJD_DEV uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

SJD_DEV float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
// round to nearest even
SJD_DEV uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// v ~= hi + lo with hi = bf16(v), lo = bf16(v - hi): about 16 significant
// bits carried in two bf16 MFMA operands.
SJD_DEV void split_bf16(float v, uint16_t& hi, uint16_t& lo) {
  hi = f32_to_bf16(v);
  lo = f32_to_bf16(v - bf16_to_f32(hi));
}

// split_bf16 for values known to be finite (no NaN / Inf handling)
SJD_DEV void split_bf16_finite(float v, uint16_t& hi, uint16_t& lo) {
  const uint32_t u = __float_as_uint(v);
  hi = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
  const float r = v - __uint_as_float((uint32_t)hi << 16);
  const uint32_t ur = __float_as_uint(r);
  lo = (uint16_t)((ur + 0x7FFFu + ((ur >> 16) & 1u)) >> 16);
}

// ---------------------------------------------------------------- reductions
SJD_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
SJD_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
SJD_DEV double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
SJD_DEV int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
SJD_DEV uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)v, o, kWave);
    uint32_t hi = __shfl_xor((uint32_t)(v >> 32), o, kWave);
    uint64_t w = ((uint64_t)hi << 32) | lo;
    v = w < v ? w : v;
  }
  return v;
}
// inclusive prefix sum within the wave
SJD_DEV int wave_incl_scan(int v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int t = __shfl_up(v, o, kWave);
    if (lane >= o) v += t;
  }
  return v;
}


// --------------------------------------------- DPP reductions (all lanes on)
// Cross-lane steps through DPP instead of the LDS permute network: within
// each 16-lane row by quad permutations and mirrors, across the four rows by
// reading lanes 0, 16, 32 and 48 (the results are wave-uniform). Every lane
// of the wave must be active: a lane outside the exec mask would feed stale
// data into its neighbours.
namespace dpp {
enum : int { kXor1 = 0xB1, kXor2 = 0x4E, kHalfMirror = 0x141, kMirror = 0x140, kShr1 = 0x111, kShr2 = 0x112,
             kShr4 = 0x114, kShr8 = 0x118, kBcast15 = 0x142, kBcast31 = 0x143 };
template <int CTRL, int ROWS = 0xF>
SJD_DEV uint32_t mov(uint32_t v) { return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xF, false); }
SJD_DEV uint32_t lane(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }
}  // namespace dpp

// op over each 16-lane row, the result in every lane of the row
template <class T, class Op>
SJD_DEV T row_reduce32(T v, Op op) {
  static_assert(sizeof(T) == 4, "32-bit payload");
  auto step = [&](uint32_t u) { return __builtin_bit_cast(T, u); };
  v = op(v, step(dpp::mov<dpp::kXor1>(__builtin_bit_cast(uint32_t, v))));
  v = op(v, step(dpp::mov<dpp::kXor2>(__builtin_bit_cast(uint32_t, v))));
  v = op(v, step(dpp::mov<dpp::kHalfMirror>(__builtin_bit_cast(uint32_t, v))));
  v = op(v, step(dpp::mov<dpp::kMirror>(__builtin_bit_cast(uint32_t, v))));
  return v;
}
template <class T, class Op>
SJD_DEV T wave_reduce32(T v, Op op) {
  v = row_reduce32(v, op);
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  const T a = __builtin_bit_cast(T, dpp::lane(u, 0)), b = __builtin_bit_cast(T, dpp::lane(u, 16));
  const T c = __builtin_bit_cast(T, dpp::lane(u, 32)), d = __builtin_bit_cast(T, dpp::lane(u, 48));
  return op(op(a, b), op(c, d));
}
// 64-bit payloads move as two 32-bit halves
template <int CTRL>
SJD_DEV uint64_t mov64(uint64_t v) {
  return ((uint64_t)dpp::mov<CTRL>((uint32_t)(v >> 32)) << 32) | dpp::mov<CTRL>((uint32_t)v);
}
template <class T, class Op>
SJD_DEV T wave_reduce64(T v, Op op) {
  static_assert(sizeof(T) == 8, "64-bit payload");
  auto as = [](uint64_t u) { return __builtin_bit_cast(T, u); };
  auto bits = [](T x) { return __builtin_bit_cast(uint64_t, x); };
  v = op(v, as(mov64<dpp::kXor1>(bits(v))));
  v = op(v, as(mov64<dpp::kXor2>(bits(v))));
  v = op(v, as(mov64<dpp::kHalfMirror>(bits(v))));
  v = op(v, as(mov64<dpp::kMirror>(bits(v))));
  const uint64_t u = bits(v);
  auto at = [&](int l) { return as(((uint64_t)dpp::lane((uint32_t)(u >> 32), l) << 32) | dpp::lane((uint32_t)u, l)); };
  return op(op(at(0), at(16)), op(at(32), at(48)));
}
SJD_DEV float wave_max_dpp(float v) { return wave_reduce32(v, [](float a, float b) { return fmaxf(a, b); }); }
SJD_DEV double wave_sum_d_dpp(double v) { return wave_reduce64(v, [](double a, double b) { return a + b; }); }
SJD_DEV uint64_t wave_min_u64_dpp(uint64_t v) {
  return wave_reduce64(v, [](uint64_t a, uint64_t b) { return a < b ? a : b; });
}
// inclusive prefix sum over the wave (lane order)
SJD_DEV int wave_incl_scan_dpp(int v) {
  v += (int)dpp::mov<dpp::kShr1>((uint32_t)v);
  v += (int)dpp::mov<dpp::kShr2>((uint32_t)v);
  v += (int)dpp::mov<dpp::kShr4>((uint32_t)v);
  v += (int)dpp::mov<dpp::kShr8>((uint32_t)v);
  v += (int)dpp::mov<dpp::kBcast15, 0xA>((uint32_t)v);
  v += (int)dpp::mov<dpp::kBcast31, 0xC>((uint32_t)v);
  return v;
}
// OR over each aligned group of 8 lanes, the result in every lane of the group
SJD_DEV uint32_t or8_dpp(uint32_t v) {
  v |= dpp::mov<dpp::kXor1>(v);
  v |= dpp::mov<dpp::kXor2>(v);
  v |= dpp::mov<dpp::kHalfMirror>(v);
  return v;
}

}  // namespace sjd
