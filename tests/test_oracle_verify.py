"""Pins for the oracle's verification step (one SJD-PAC iteration, Alg. 1).

Each check is fixed by the paper or by mathematics, not by the oracle:
- top-k / temperature softmax against an independent library (torch) and a
  lexsort statement of the tie order;
- Rejection Sampling Lemma / Theorem 1 (Appendix A): committed token ~ p for
  any draft law q, acceptance probability sum_x min(p, q) = 1 - TV(p, q)
  (Sec. 4.2);
- Theorem 2 (Appendix A.3): K candidates drawn without replacement from q and
  verified against p^(k), q^(k) still give a token ~ p;
- all drafts accepted when p = q (ratio 1 in the accept test of Alg. 1);
- a chain window of independent rows has E[n_c] = sum_i prod_{j<i-1} a_j;
- with L = 1 the step is one plain autoregressive draw (n_c = 1).
"""
import numpy as np
import pytest
import torch
from scipy import stats


def softmax_topk_np(l, top_k, T=1.0):
    l = np.asarray(l, np.float64)
    V = l.size
    k = V if top_k <= 0 or top_k >= V else top_k
    order = np.lexsort((np.arange(V), -l))[:k]
    z = np.full(V, -np.inf)
    z[order] = (l[order] - l[order].max()) / T
    p = np.exp(z)
    return p / p.sum()


def chi2_p(counts, probs):
    counts = np.asarray(counts, float)
    exp = np.asarray(probs, float) * counts.sum()
    m = exp > 1e-12
    assert counts[~m].sum() == 0, "mass where the target law has none"
    if m.sum() == 1:
        return 1.0
    return stats.chi2.sf(((counts[m] - exp[m]) ** 2 / exp[m]).sum(), m.sum() - 1)


def sample_rows(rng, probs, n):
    """n independent draws from each row of probs (numpy, inverse CDF)."""
    c = np.cumsum(probs, axis=-1)
    c[..., -1] = 1.0
    u = rng.random((n,) + probs.shape[:-1])
    return (u[..., None] > c).sum(-1)


def draw_without_replacement(rng, q, k, n):
    """n ordered draws of k distinct tokens from q (successive sampling)."""
    out = np.zeros((n, k), np.int64)
    w = np.tile(q, (n, 1)).astype(np.float64)
    for i in range(k):
        s = w.sum(1, keepdims=True)
        c = np.cumsum(w / s, 1)
        c[:, -1] = 1.0
        x = (rng.random((n, 1)) > c).sum(1)
        out[:, i] = x
        w[np.arange(n), x] = 0.0
    return out


# ----------------------------------------------------------------------------- top-k softmax

@pytest.mark.parametrize("V,top_k,T", [(50, 10, 1.0), (50, 0, 1.0), (50, 1, 1.0), (50, 49, 0.7),
                                       (50, 50, 1.3), (50, 77, 1.0), (1, 0, 1.0), (4096, 2000, 1.0)])
def test_topk_softmax_vs_torch(orc, V, top_k, T):
    rng = np.random.default_rng(V * 31 + top_k)
    l = (rng.standard_normal(V) * 2).astype(np.float32)
    p = orc.topk_softmax(l, top_k, T)
    k = V if top_k <= 0 or top_k >= V else top_k
    t = torch.from_numpy(l).double()
    vals, idx = torch.topk(t, k)
    ref = torch.zeros(V, dtype=torch.float64)
    ref[idx] = torch.softmax((vals - vals.max()) / T, 0)
    assert np.abs(p - ref.numpy()).max() < 2e-7
    assert ((p > 0).sum()) == k
    assert abs(p.astype(np.float64).sum() - 1) < 1e-5


def test_topk_tie_order(orc):
    # many equal logits: the set is taken by (value desc, index asc)
    l = np.array([1, 3, 3, 2, 3, 3, 0, 3], np.float32)
    p = orc.topk_softmax(l, 3)
    assert np.nonzero(p)[0].tolist() == [1, 2, 4]
    ref = softmax_topk_np(l, 3)
    assert np.abs(p - ref).max() < 1e-7


def test_topk_minus_inf_entries(orc):
    l = np.array([0.0, -np.inf, 1.0, -np.inf], np.float32)
    p = orc.topk_softmax(l, 0)
    assert p[1] == 0 and p[3] == 0
    assert abs(p[2] / p[0] - np.e) < 1e-5


# ----------------------------------------------------------------------------- single draft

def _single_row_case(orc, lp, lq, n, seed, top_k=0):
    V = lp.size
    rng = np.random.default_rng(seed)
    p = softmax_topk_np(lp, top_k)
    q = softmax_topk_np(lq, top_k)
    drafts = sample_rows(rng, q[None, :], n)[:, 0]
    cur = np.broadcast_to(lp, (n, 1, V))
    dr = np.broadcast_to(lq, (n, 1, V))
    meta = np.tile(np.array([0, 1, 0, 0], np.int32), (n, 1))
    out = orc.verify(cur, dr, drafts[:, None], meta, K=1, D=0, top_k=top_k, seed=seed)
    assert (out["meta"][:, 0] == 1).all()
    tok = out["tok"][:, 0]
    acc = out["rows"][:, 0, 1] == 1
    return p, q, tok, acc, drafts


CASES = {
    "random": (np.array([0.3, -1.0, 2.0, 0.1, 0.5, -0.2]), np.array([1.0, 0.2, -0.5, 0.0, 1.5, -2.0])),
    "equal": (np.array([0.3, -1.0, 2.0, 0.1, 0.5, -0.2]), np.array([0.3, -1.0, 2.0, 0.1, 0.5, -0.2])),
    "disjoint": (np.array([0.0, 0.0, 0.0, -np.inf, -np.inf, -np.inf]),
                 np.array([-np.inf, -np.inf, -np.inf, 0.0, 1.0, 2.0])),
    "q_zeros": (np.array([0.5, 0.1, 0.2, 1.0, -1.0, 0.0]), np.array([2.0, -np.inf, 1.0, -np.inf, 0.0, -np.inf])),
    "peaked": (np.array([8.0, 0.0, 0.0, 0.0, 0.0, 0.0]), np.array([0.0, 0.0, 0.0, 0.0, 0.0, 8.0])),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_single_draft_lossless_and_acceptance(orc, case):
    lp, lq = (a.astype(np.float32) for a in CASES[case])
    n = 1_000_000
    p, q, tok, acc, drafts = _single_row_case(orc, lp, lq, n, seed=sum(map(ord, case)))
    counts = np.bincount(tok, minlength=p.size)
    assert chi2_p(counts, p) > 1e-4
    a = np.minimum(p, q).sum()  # 1 - TV(p, q)
    k = int(acc.sum())
    ci = stats.binomtest(k, n).proportion_ci(confidence_level=0.9999)
    assert ci.low <= a <= ci.high, (k / n, a)
    # accepted tokens are the drafts, rejected ones come from max(0, p - q)
    assert (tok[acc] == drafts[acc]).all()
    r = np.maximum(p - q, 0)
    if r.sum() > 0 and (~acc).sum() > 0:
        assert chi2_p(np.bincount(tok[~acc], minlength=p.size), r / r.sum()) > 1e-4


def test_single_draft_with_topk_and_temperature(orc):
    rng = np.random.default_rng(5)
    lp = (rng.standard_normal(8) * 2).astype(np.float32)
    lq = (lp + rng.standard_normal(8)).astype(np.float32)
    n = 1_000_000
    V = 8
    for top_k, T in [(4, 1.0), (5, 0.6)]:
        p = softmax_topk_np(lp, top_k, T)
        q = softmax_topk_np(lq, top_k, T)
        drafts = sample_rows(rng, q[None, :], n)[:, 0]
        meta = np.tile(np.array([0, 1, 0, 0], np.int32), (n, 1))
        out = orc.verify(np.broadcast_to(lp, (n, 1, V)), np.broadcast_to(lq, (n, 1, V)), drafts[:, None],
                         meta, K=1, D=0, top_k=top_k, T=T, seed=top_k)
        assert chi2_p(np.bincount(out["tok"][:, 0], minlength=V), p) > 1e-4


# ----------------------------------------------------------------------------- K candidates

@pytest.mark.parametrize("K", [2, 3, 4])
def test_k_candidates_without_replacement_lossless(orc, K):
    V = 6
    rng = np.random.default_rng(100 + K)
    lp = np.array([0.3, -1.0, 2.0, 0.1, 0.5, -0.2], np.float32)
    lq = np.array([1.0, 0.2, -0.5, 0.0, 1.5, -2.0], np.float32)
    p, q = softmax_topk_np(lp, 0), softmax_topk_np(lq, 0)
    n = 1_000_000
    cand = draw_without_replacement(rng, q, K, n)
    L = K  # one tree row (depth 0) plus K - 1 sibling rows
    cur = np.zeros((n, L, V), np.float32)
    cur[:, 0] = lp
    sib_logits = (rng.standard_normal((K - 1, V)) * 1.5).astype(np.float32)
    cur[:, 1:] = sib_logits
    dr = np.zeros((n, L, V), np.float32)
    dr[:, 0] = lq
    draft_tok = np.zeros((n, L), np.int32)
    draft_tok[:, 0] = cand[:, 0]
    sib = cand[:, 1:].reshape(n, 1, K - 1).astype(np.int32)
    meta = np.tile(np.array([1, 1, 0, 0], np.int32), (n, 1))
    out = orc.verify(cur, dr, draft_tok, meta, K=K, D=1, top_k=0, sib=sib, seed=K)
    tok0 = out["tok"][:, 0]
    assert chi2_p(np.bincount(tok0, minlength=V), p) > 1e-4
    stage = out["rows"][:, 0, 1]
    nc = out["meta"][:, 0]
    # candidate 1 accepted with probability sum min(p, q) (plain rejection test)
    a = np.minimum(p, q).sum()
    ci = stats.binomtest(int((stage == 1).sum()), n).proportion_ci(confidence_level=0.9999)
    assert ci.low <= a <= ci.high
    # an accepted sibling commits itself plus a bonus token drawn from its own row
    sib_acc = stage >= 2
    assert (nc[sib_acc] == 2).all() and (nc[~sib_acc] == 1).all()
    assert (out["meta"][sib_acc, 5] == stage[sib_acc]).all()
    for k in range(2, K + 1):
        m = stage == k
        assert (tok0[m] == cand[m, k - 1]).all()
        if m.sum() > 2000:
            pb = softmax_topk_np(sib_logits[k - 2], 0)
            assert chi2_p(np.bincount(out["tok"][m, 1], minlength=V), pb) > 1e-4


# ----------------------------------------------------------------------------- window-level

def _chain_window(orc, rng, n, L, V, noise, top_k=0, identical=False):
    lp = (rng.standard_normal((L, V)) * 2).astype(np.float32)
    lq = lp.copy() if identical else (lp + rng.standard_normal((L, V)) * noise).astype(np.float32)
    q = np.stack([softmax_topk_np(r, top_k) for r in lq])
    p = np.stack([softmax_topk_np(r, top_k) for r in lp])
    drafts = sample_rows(rng, q, n).astype(np.int32)
    meta = np.tile(np.array([0, L, 0, 0], np.int32), (n, 1))
    out = orc.verify(np.broadcast_to(lp, (n, L, V)), np.broadcast_to(lq, (n, L, V)), drafts, meta,
                     K=4, D=min(3, L // 4), top_k=top_k, seed=11)
    return p, q, drafts, out


def test_all_accept_when_p_equals_q(orc):
    rng = np.random.default_rng(3)
    n, L, V = 2000, 16, 64
    p, q, drafts, out = _chain_window(orc, rng, n, L, V, 0.0, top_k=20, identical=True)
    assert (out["meta"][:, 0] == L).all()
    assert (out["meta"][:, 1] == -1).all()
    assert (out["tok"] == drafts).all()
    # nothing rejected: no proactive drafting, the whole next window is appended
    assert (out["meta"][:, 2] == 0).all() and (out["meta"][:, 4] == 0).all()


def test_chain_expected_accept_length_closed_form(orc):
    rng = np.random.default_rng(4)
    n, L, V = 200_000, 8, 12
    p, q, drafts, out = _chain_window(orc, rng, n, L, V, 0.6)
    a = np.minimum(p, q).sum(1)
    # E[n_c] = sum_{i=1}^{L} P(rows 0..i-2 accepted)
    expect = sum(np.prod(a[: i - 1]) for i in range(1, L + 1))
    nc = out["meta"][:, 0].astype(float)
    se = nc.std() / np.sqrt(n)
    assert abs(nc.mean() - expect) < 5 * se, (nc.mean(), expect, se)
    # each committed position is distributed as its target row
    r = out["meta"][:, 1]
    for j in range(3):
        m = (r == -1) | (r >= j)
        assert chi2_p(np.bincount(out["tok"][m, j], minlength=V), p[j]) > 1e-4


def test_single_slot_window_is_plain_ar(orc):
    """L = 1: one slot, no draft distribution, one committed token per step,
    drawn from p by the stage-0 race of that row."""
    rng = np.random.default_rng(8)
    n, V = 1_000_000, 7
    lp = (rng.standard_normal(V) * 1.5).astype(np.float32)
    meta = np.tile(np.array([0, 0, 0, 0], np.int32), (n, 1))
    dummy = np.zeros((n, 1), np.int32)
    out = orc.verify(np.broadcast_to(lp, (n, 1, V)), np.broadcast_to(lp, (n, 1, V)), dummy, meta,
                     K=4, D=0, top_k=0, seed=21, step=4)
    assert (out["meta"][:, 0] == 1).all()
    p = softmax_topk_np(lp, 0)
    assert chi2_p(np.bincount(out["tok"][:, 0], minlength=V), p) > 1e-4
    for b in range(0, n, 50000):
        x, _ = orc.race(orc.topk_softmax(lp, 0), 21, orc.TAG_RES, 0, 0, b, 4)
        assert out["tok"][b, 0] == x


def test_next_window_structure_with_pd(orc):
    rng = np.random.default_rng(12)
    n, L, V, K, D = 3000, 16, 40, 4, 3
    p, q, drafts, out = _chain_window(orc, rng, n, L, V, 2.0, top_k=25)
    for b in range(n):
        m = out["meta"][b]
        n_c, r, Dn, ns2, nq2 = m[:5]
        assert 1 <= n_c <= L
        if r >= 0:
            assert n_c == r + 1
            assert Dn == min(D, L - n_c, L // K)
        else:
            assert n_c == L and Dn == 0
        assert ns2 == L - (K - 1) * Dn
        assert nq2 == max(0, min(ns2, L - n_c))
        nxt = out["next"][b]
        assert (nxt[:ns2] >= 0).all() and (nxt[:ns2] < V).all() and (nxt[ns2:] == -1).all()
        # the drafts carried over are the row outcomes after the commit point
        rows = out["rows"][b, :, 0]
        assert (nxt[:nq2] == rows[n_c:n_c + nq2]).all()
        for d in range(Dn):
            sib = out["sib"][b, d]
            j = n_c + d
            live = sib[sib >= 0]
            assert len(set(live.tolist())) == len(live)
            assert rows[j] not in live.tolist()
            assert (p[j][live] > 0).all()


def test_forced_row_end_tokens(orc):
    """Row-end positions (generated index g with g mod (W+1) == W) take the row
    end token, count as accepted and get no siblings."""
    rng = np.random.default_rng(13)
    n, L, V, W = 500, 12, 30, 3
    eol = 1000
    lp = (rng.standard_normal((n, L, V)) * 2).astype(np.float32)
    lq = (lp + rng.standard_normal((n, L, V)) * 3).astype(np.float32)
    g0 = rng.integers(0, 50, n)
    drafts = rng.integers(0, V, (n, L)).astype(np.int32)
    forced = ((g0[:, None] + np.arange(L)) % (W + 1)) == W
    drafts[forced] = eol
    meta = np.stack([np.zeros(n), np.full(n, L), g0, np.zeros(n)], 1).astype(np.int32)
    out = orc.verify(lp, lq, drafts, meta, K=4, D=3, top_k=10, seed=3, eol_id=eol, row_len=W)
    for b in range(n):
        n_c, r = out["meta"][b, :2]
        rows = out["rows"][b]
        for j in range(L):
            if forced[b, j]:
                assert rows[j, 0] == eol and rows[j, 1] == -1
                assert r != j
        for i in range(n_c):
            if forced[b, i]:
                assert out["tok"][b, i] == eol
        ns2 = out["meta"][b, 3]
        gn = g0[b] + n_c
        for i in range(ns2):
            if (gn + i) % (W + 1) == W:
                assert out["next"][b, i] == eol
        for d in range(out["meta"][b, 2]):
            if (gn + d) % (W + 1) == W:
                assert (out["sib"][b, d] == -1).all()
        assert out["meta"][b, 6] == g0[b] + n_c


def test_vanilla_sjd_tail_is_fresh(orc):
    """AC off (Sec. 3.3): rows after the first rejection are redrawn from their
    target rows, independently of the old drafts."""
    rng = np.random.default_rng(14)
    n, L, V = 1_000_000, 4, 5
    lp = (rng.standard_normal((L, V)) * 1.5).astype(np.float32)
    lq = (lp + rng.standard_normal((L, V)) * 2.0).astype(np.float32)
    p = np.stack([softmax_topk_np(r, 0) for r in lp])
    q = np.stack([softmax_topk_np(r, 0) for r in lq])
    drafts = sample_rows(rng, q, n).astype(np.int32)
    meta = np.tile(np.array([0, L, 0, 0], np.int32), (n, 1))
    out = orc.verify(np.broadcast_to(lp, (n, L, V)), np.broadcast_to(lq, (n, L, V)), drafts, meta,
                     K=1, D=0, top_k=0, flags=0, seed=5)
    r = out["meta"][:, 1]
    m = r == 0  # rejected at row 0: next drafts are rows 1..3, fresh from p
    assert chi2_p(np.bincount(out["next"][m, 0], minlength=V), p[1]) > 1e-4
    # independent of the old draft at that row
    same = (out["next"][m, 0] == drafts[m, 1]).mean()
    assert abs(same - (p[1] * q[1]).sum()) < 5 * np.sqrt(same * (1 - same) / m.sum())


def test_verify_rejects_bad_arguments(orc):
    cur = np.zeros((1, 4, 8), np.float32)
    tok = np.zeros((1, 4), np.int32)
    with pytest.raises(ValueError):
        orc.verify(cur, cur, tok, np.array([[2, 0, 0, 0]], np.int32), K=4, D=1, top_k=0)  # K*D_in > L
    with pytest.raises(ValueError):
        orc.verify(cur, cur, tok, np.array([[0, 5, 0, 0]], np.int32), K=1, D=0, top_k=0)  # n_q > n_s
    with pytest.raises(ValueError):
        orc.verify(cur, cur, tok, np.array([[0, 0, 0, 0]], np.int32), K=1, D=0, top_k=0, T=0.0)
