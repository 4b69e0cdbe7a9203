/* Oracle: counter-based random numbers and the exponential race sampler.
 *
 * Test infrastructure only (see oracle.h); shares no code with the HIP path.
 *
 * Philox4x32-10 follows its publication (Salmon, Moraes, Dror, Shaw, SC'11):
 * each round multiplies counter words 0 and 2 by two fixed odd constants,
 * takes the 64-bit products apart into high and low halves, and forms the new
 * counter as (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the two key words are
 * bumped by the Weyl constants (golden ratio, sqrt(3) - 1) between rounds.
 *
 * The paper does not say how its "Sample" step draws a token (Alg. 1, the
 * reject branch); the oracle uses the exponential race, whose winner has law
 * w_x / sum(w) for any non-negative weights (so an unnormalised residual
 * max(0, p - q) needs no normalisation), and whose K smallest keys are a draw
 * of K tokens without replacement (the successive-sampling law that the
 * paper's Theorem 2 uses for q^(k)).
 */
#include "oracle.h"

#include <math.h>
#include <stddef.h>

static const uint32_t PHILOX_M0 = 0xD2511F53u;
static const uint32_t PHILOX_M1 = 0xCD9E8D57u;
static const uint32_t PHILOX_W0 = 0x9E3779B9u;
static const uint32_t PHILOX_W1 = 0xBB67AE85u;

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    uint64_t prod0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
    uint64_t prod1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
    uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
    uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    uint32_t n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

uint32_t orc_bits(uint64_t seed, uint32_t tag, uint32_t stage, uint32_t row,
                  uint32_t trial, uint32_t step, uint32_t x) {
  uint32_t ctr[4] = {x >> 2, trial, (tag << 24) | ((stage & 0xFFu) << 16) | (row & 0xFFFFu), step};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t out[4];
  orc_philox4x32_10(ctr, key, out);
  return out[x & 3u];
}

float orc_uniform(uint32_t bits) { return (float)(bits >> 8) * 0x1p-24f; }

float orc_exp1(uint32_t bits) {
  float one_minus_u = 1.0f - orc_uniform(bits); /* exact: u is a multiple of 2^-24 */
  return -logf(one_minus_u);
}

int orc_race(const float* w, int V, uint64_t seed, uint32_t tag, uint32_t stage,
             uint32_t row, uint32_t trial, uint32_t step, float* gap) {
  return orc_race_ranked(w, NULL, V, seed, tag, stage, row, trial, step, gap);
}

int orc_race_ranked(const float* w, const int* rank, int V, uint64_t seed, uint32_t tag, uint32_t stage,
                    uint32_t row, uint32_t trial, uint32_t step, float* gap) {
  int best = -1;
  float best_key = INFINITY, second_key = INFINITY;
  for (int x = 0; x < V; ++x) {
    if (!(w[x] > 0.0f)) continue;
    const uint32_t e_idx = rank ? (uint32_t)rank[x] : (uint32_t)x;
    float e = orc_exp1(orc_bits(seed, tag, stage, row, trial, step, e_idx));
    float key = e / w[x];
    if (best < 0 || key < best_key) {
      second_key = best_key;
      best_key = key;
      best = x;
    } else if (key < second_key) {
      second_key = key;
    }
  }
  if (gap) {
    if (best < 0 || !isfinite(second_key)) *gap = 1.0f;
    else if (second_key <= 0.0f) *gap = 0.0f;
    else *gap = (second_key - best_key) / second_key;
  }
  return best;
}

int orc_race_topn(const float* w, int V, int n, int excl, uint64_t seed, uint32_t tag,
                  uint32_t stage, uint32_t row, uint32_t trial, uint32_t step, int* out,
                  float* gap) {
  return orc_race_topn_ranked(w, NULL, V, n, excl, seed, tag, stage, row, trial, step, out, gap);
}

int orc_race_topn_ranked(const float* w, const int* rank, int V, int n, int excl, uint64_t seed,
                         uint32_t tag, uint32_t stage, uint32_t row, uint32_t trial, uint32_t step,
                         int* out, float* gap) {
  /* keeps the n + 1 smallest (key, index) pairs, in ascending key order with
   * ties to the smaller index, by insertion */
  float keys[17];
  int idx[17];
  int have = 0;
  if (n < 0 || n > 16) return -1;
  const int cap = n + 1;
  for (int x = 0; x < V; ++x) {
    if (x == excl || !(w[x] > 0.0f)) continue;
    const uint32_t e_idx = rank ? (uint32_t)rank[x] : (uint32_t)x;
    float key = orc_exp1(orc_bits(seed, tag, stage, row, trial, step, e_idx)) / w[x];
    if (have == cap && !(key < keys[cap - 1])) continue;
    int pos = have < cap ? have : cap - 1;
    while (pos > 0 && key < keys[pos - 1]) {
      keys[pos] = keys[pos - 1];
      idx[pos] = idx[pos - 1];
      --pos;
    }
    keys[pos] = key;
    idx[pos] = x;
    if (have < cap) ++have;
  }
  float g = INFINITY;
  for (int i = 0; i + 1 < have; ++i) {
    float rel = keys[i + 1] > 0.0f ? (keys[i + 1] - keys[i]) / keys[i + 1] : 0.0f;
    if (rel < g) g = rel;
  }
  if (gap) *gap = g;
  int got = have < n ? have : n;
  for (int i = 0; i < n; ++i) out[i] = i < got ? idx[i] : -1;
  return got;
}

void orc_race_many(const float* w, int V, int n, uint64_t seed, uint32_t tag, uint32_t stage,
                   uint32_t row, uint32_t step, int trials, int* out) {
  orc_race_many_ranked(w, NULL, V, n, seed, tag, stage, row, step, trials, out);
}

void orc_race_many_ranked(const float* w, const int* rank, int V, int n, uint64_t seed, uint32_t tag,
                          uint32_t stage, uint32_t row, uint32_t step, int trials, int* out) {
#pragma omp parallel for schedule(static)
  for (int b = 0; b < trials; ++b) {
    if (n <= 1) out[b] = orc_race_ranked(w, rank, V, seed, tag, stage, row, (uint32_t)b, step, NULL);
    else orc_race_topn_ranked(w, rank, V, n, -1, seed, tag, stage, row, (uint32_t)b, step,
                              out + (size_t)b * n, NULL);
  }
}
