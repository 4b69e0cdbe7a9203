"""Pins for the oracle's random numbers and race sampler.

- Philox4x32-10 against the published known-answer vectors of its reference
  implementation and against an independent implementation (ROCm's rocRAND
  header, compiled for the host).
- The exponential race: the winner's law is w / sum(w); the n smallest keys
  are an ordered draw without replacement whose tuple law is the product of
  successive renormalised weights (the q^(k) of the paper's Theorem 2).
"""
import itertools
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(t, 16) for t in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_philox_known_answers(orc):
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, want in rows:
        assert orc.philox(ctr, key) == want


ROCRAND_PROG = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
int main() {
  unsigned long long seed, x, y, z, w, lane;
  while (std::scanf("%llu %llu %llu %llu %llu %llu", &seed, &x, &y, &z, &w, &lane) == 6) {
    unsigned long long subseq = z | (w << 32);
    unsigned long long offset = 4ull * (x | (y << 32)) + lane;
    rocrand_device::philox4x32_10_engine e(seed, subseq, offset);
    std::printf("%u\n", e());
  }
  return 0;
}
"""


def test_philox_matches_rocrand(orc, tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("rocRAND header / hipcc not available")
    src = tmp_path / "rr.cpp"
    src.write_text(ROCRAND_PROG)
    exe = tmp_path / "rr"
    subprocess.run([hipcc, "-O1", str(src), "-o", str(exe)], check=True, capture_output=True)
    rng = np.random.default_rng(123)
    cases = []
    for _ in range(200):
        seed = int(rng.integers(0, 2**63))
        x = int(rng.integers(0, 2**32))
        y = int(rng.integers(0, 2**29))
        z = int(rng.integers(0, 2**32))
        w = int(rng.integers(0, 2**31))
        lane = int(rng.integers(0, 4))
        cases.append((seed, x, y, z, w, lane))
    inp = "\n".join(" ".join(str(v) for v in c) for c in cases) + "\n"
    res = subprocess.run([str(exe)], input=inp, capture_output=True, text=True, check=True)
    got = [int(t) for t in res.stdout.split()]
    for (seed, x, y, z, w, lane), g in zip(cases, got):
        want = orc.philox([x, y, z, w], [seed & 0xFFFFFFFF, seed >> 32])[lane]
        assert want == g


def test_stream_counter_layout(orc):
    seed = 0x1234_5678_9ABC_DEF0
    for tag, stage, row, trial, step, x in [(1, 0, 0, 0, 0, 0), (2, 3, 17, 4095, 9, 16383),
                                             (5, 0, 63, 7, 123456, 65535), (6, 0, 5, 0, 0xFFFFFFFF, 2)]:
        ctr = [x >> 2, trial, (tag << 24) | (stage << 16) | row, step]
        assert orc.bits(seed, tag, stage, row, trial, step, x) == \
            orc.philox(ctr, [seed & 0xFFFFFFFF, seed >> 32])[x & 3]


def test_uniform_grid_and_range(orc):
    assert orc.uniform(0) == 0.0
    assert orc.uniform(0xFFFFFFFF) == 1.0 - 2.0**-24
    assert orc.uniform(0x100) == 2.0**-24
    assert orc.uniform(0xFF) == 0.0


def _chi2_p(counts, probs):
    exp = probs * counts.sum()
    m = exp > 0
    assert counts[~m].sum() == 0
    if m.sum() == 1:
        return 1.0
    chi = ((counts[m] - exp[m]) ** 2 / exp[m]).sum()
    return stats.chi2.sf(chi, m.sum() - 1)


@pytest.mark.parametrize("w", [[0.1, 0.2, 0.3, 0.4, 0.0], [1.0, 1.0, 1.0, 1.0, 1.0],
                               [5e-3, 7.0, 0.25, 3.0, 1e-1], [0.0, 0.0, 2.0, 0.0, 0.0]])
def test_race_winner_law(orc, w):
    w = np.array(w, np.float32)
    n = 1_000_000
    win = orc.race_many(w, 1, n, seed=77, tag=orc.TAG_RES, stage=1, row=3, step=5)
    counts = np.bincount(win, minlength=w.size).astype(float)
    p = w.astype(np.float64) / w.sum()
    assert _chi2_p(counts, p) > 1e-4


def test_race_topn_tuple_law(orc):
    """Ordered draws of 3 from 5 without replacement: P(c1,c2,c3) =
    w1/S * w2/(S-w1) * w3/(S-w1-w2) (successive sampling), 60 tuples."""
    w = np.array([0.05, 0.4, 0.15, 0.3, 0.1], np.float32)
    n = 1_000_000
    draws = orc.race_many(w, 3, n, seed=9, tag=orc.TAG_PD, stage=0, row=1, step=2)
    tuples = list(itertools.permutations(range(5), 3))
    index = {t: i for i, t in enumerate(tuples)}
    code = draws[:, 0] * 25 + draws[:, 1] * 5 + draws[:, 2]
    lut = np.full(125, -1)
    for t, i in index.items():
        lut[t[0] * 25 + t[1] * 5 + t[2]] = i
    ids = lut[code]
    assert (ids >= 0).all()
    counts = np.bincount(ids, minlength=len(tuples)).astype(float)
    wd = w.astype(np.float64)
    S = wd.sum()
    probs = np.array([wd[a] / S * wd[b] / (S - wd[a]) * wd[c] / (S - wd[a] - wd[b]) for a, b, c in tuples])
    assert abs(probs.sum() - 1) < 1e-12
    assert _chi2_p(counts, probs) > 1e-4


# Ranked races: the verification step draws one stream element per kept
# (top-k) token, element rank[x] for token x, its position among the kept
# tokens in index order. The ranks are a bijection from the kept tokens onto
# elements 0 .. k-1, all independent uniforms, so the laws must be the
# unranked ones; pinned here with a non-identity rank (a kept subset of a
# larger vocabulary).
KEPT = np.array([2, 3, 7, 8, 11, 15])


def _ranked(weights, V=16):
    w = np.zeros(V, np.float32)
    w[KEPT[:len(weights)]] = weights
    rank = np.full(V, -1, np.int32)
    rank[KEPT[:len(weights)]] = np.arange(len(weights))
    return w, rank


def test_ranked_race_winner_law(orc):
    w, rank = _ranked([0.3, 1.2, 0.05, 2.0, 0.7, 0.4])
    n = 1_000_000
    win = orc.race_many_ranked(w, rank, 1, n, seed=31, tag=orc.TAG_RES, stage=2, row=5, step=9)
    counts = np.bincount(win, minlength=w.size).astype(float)
    assert _chi2_p(counts, w.astype(np.float64) / w.sum()) > 1e-4


def test_ranked_race_topn_tuple_law(orc):
    """Ordered draws of 3 from the 5 kept tokens without replacement
    (successive sampling), 60 tuples."""
    w, rank = _ranked([0.05, 0.4, 0.15, 0.3, 0.1])
    kept = KEPT[:5]
    n = 1_000_000
    draws = orc.race_many_ranked(w, rank, 3, n, seed=12, tag=orc.TAG_PD, stage=0, row=4, step=3)
    pos = np.full(w.size, -1)
    pos[kept] = np.arange(5)
    d = pos[draws]
    assert (d >= 0).all()
    tuples = list(itertools.permutations(range(5), 3))
    lut = np.full(125, -1)
    for i, t in enumerate(tuples):
        lut[t[0] * 25 + t[1] * 5 + t[2]] = i
    ids = lut[d[:, 0] * 25 + d[:, 1] * 5 + d[:, 2]]
    assert (ids >= 0).all()
    counts = np.bincount(ids, minlength=len(tuples)).astype(float)
    wd = w[kept].astype(np.float64)
    S = wd.sum()
    probs = np.array([wd[a] / S * wd[b] / (S - wd[a]) * wd[c] / (S - wd[a] - wd[b]) for a, b, c in tuples])
    assert _chi2_p(counts, probs) > 1e-4


def test_ranked_race_is_the_race_over_the_compact_list(orc):
    """Element rank[x] of the stream for token x: the ranked race over the
    vocabulary picks the token the plain race over the compacted kept list
    picks (same keys), and the ranked draws without replacement exclude a
    token by vocabulary id."""
    w, rank = _ranked([0.3, 1.2, 0.05, 2.0, 0.7, 0.4])
    wc = w[KEPT]
    for trial in range(200):
        x, g1 = orc.race_ranked(w, rank, 5, orc.TAG_BONUS, 1, 2, trial, 7)
        y, g2 = orc.race(wc, 5, orc.TAG_BONUS, 1, 2, trial, 7)
        assert x == KEPT[y] and g1 == g2
        top, _ = orc.race_topn_ranked(w, rank, 3, int(KEPT[1]), 5, orc.TAG_PD, 0, 2, trial, 7)
        assert KEPT[1] not in top.tolist() and len(set(top.tolist())) == 3


def test_race_topn_exclusion_and_padding(orc):
    w = np.array([0.0, 1.0, 2.0, 0.0, 3.0], np.float32)
    out, _ = orc.race_topn(w, 4, 2, 1, orc.TAG_PD, 0, 0, 0, 0)
    # only tokens 1 and 4 remain (0, 3 have no weight, 2 excluded)
    assert sorted(out[:2].tolist()) == [1, 4] and out[2:].tolist() == [-1, -1]


def test_race_ties_go_to_smaller_index(orc):
    # identical weights and, for x in one Philox block, distinct keys; an
    # all-infinite key set (tiny weights) ties everywhere and must pick x = 0
    w = np.full(8, 1e-45, np.float32)
    x, _ = orc.race(w, 0, orc.TAG_RES, 0, 0, 0, 0)
    assert x == 0
