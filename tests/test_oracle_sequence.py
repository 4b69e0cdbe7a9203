"""Sequence-level pins for the whole oracle step: the paper's losslessness
claim (SJD-PAC is rigorously lossless, Sec. 4.3 and Appendix A) checked by
brute force on a tabular toy model whose logits hash the entire context, so
any slip in context, commit, KV bookkeeping, AC, PD, bonus or placeholder
handling changes the law of the generated sequence.

The exact autoregressive joint law is computed here with numpy from the toy
model's logits alone (no oracle sampling code), and the histogram of 200k-400k
generated sequences is compared with it by a chi-square test.

Also: greedy decoding (top_k = 1) reaches the Jacobi fixed point, so the
output must equal sequential argmax decoding (Sec. 3.3).
"""
import itertools

import numpy as np
import pytest
from scipy import stats

PROMPT = [1, 2]


def toy_probs(orc, ctx, V, salt, top_k=0, T=1.0):
    l = orc.toy_logits(np.array(ctx, np.int32), V, salt).astype(np.float64)
    k = V if top_k <= 0 or top_k >= V else top_k
    order = np.lexsort((np.arange(V), -l))[:k]
    z = np.full(V, -np.inf)
    z[order] = (l[order] - l[order].max()) / T
    p = np.exp(z)
    return p / p.sum()


def exact_law(orc, N, V, salt, top_k=0, T=1.0, row_len=0, eol=-1):
    probs = np.zeros(V ** N)
    for i, seq in enumerate(itertools.product(range(V), repeat=N)):
        pr = 1.0
        ctx = list(PROMPT)
        for g, x in enumerate(seq):
            if row_len > 0 and g % (row_len + 1) == row_len:
                pr *= 1.0 if x == eol else 0.0
            else:
                pr *= toy_probs(orc, ctx, V, salt, top_k, T)[x]
            ctx.append(x)
        probs[i] = pr
    return probs


def check_law(orc, *, L, K, D, flags, runs, N=5, V=3, salt=7, top_k=0, T=1.0, row_len=0, eol=-1, seed0=1000):
    law = exact_law(orc, N, V, salt, top_k, T, row_len, eol)
    assert abs(law.sum() - 1) < 1e-9
    cfg = orc.gen_cfg(L=L, V=V, K=K, D=D, flags=flags, n_prompt=len(PROMPT), n_gen=N, toy_salt=salt,
                      top_k=top_k, T=T, row_len=row_len, eol_id=eol)
    out, steps, hist = orc.generate_many(cfg, PROMPT, runs, seed0)
    idx = np.zeros(runs, np.int64)
    for i in range(N):
        idx = idx * V + out[:, i]
    cnt = np.bincount(idx, minlength=V ** N).astype(float)
    exp = law * runs
    m = exp > 0
    assert cnt[~m].sum() == 0, "sequences of zero probability were generated"
    chi = ((cnt[m] - exp[m]) ** 2 / exp[m]).sum()
    pval = stats.chi2.sf(chi, m.sum() - 1)
    return pval, steps, hist


MODES = {"sjd": 0, "ac": 1, "pd": 2, "ac+pd": 3}


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("L,K,D", [(1, 1, 0), (2, 2, 1), (3, 2, 1), (4, 2, 2), (4, 3, 1), (5, 2, 2), (6, 3, 2)])
def test_sequence_law_equals_autoregressive(orc, mode, L, K, D):
    pval, steps, hist = check_law(orc, L=L, K=K, D=D, flags=MODES[mode], runs=1_000_000)
    assert pval > 1e-4, pval
    if L == 1:
        assert (steps == 5).all()


def test_sequence_law_larger_vocab_topk_temperature(orc):
    pval, _, _ = check_law(orc, L=4, K=3, D=1, flags=3, runs=1_000_000, N=4, V=4, salt=11, top_k=3, T=0.8)
    assert pval > 1e-4, pval


def test_sequence_law_with_forced_row_ends(orc):
    # rows of 2 image tokens followed by the row-end token 2 (inside the vocab)
    pval, _, _ = check_law(orc, L=4, K=2, D=2, flags=3, runs=1_000_000, N=6, V=3, salt=5, row_len=2, eol=2)
    assert pval > 1e-4, pval


def test_acceptance_improves_over_sjd_on_a_local_model(orc):
    """Shape check only (no paper number applies to a toy model): AC keeps
    more of the old window than the vanilla fresh tail, so the mean number of
    steps for the same output falls."""
    _, st_sjd, _ = check_law(orc, L=5, K=2, D=2, flags=0, runs=50_000, N=5, V=3)
    _, st_ac, _ = check_law(orc, L=5, K=2, D=2, flags=1, runs=50_000, N=5, V=3)
    assert st_ac.mean() <= st_sjd.mean() + 0.02


@pytest.mark.parametrize("L,K,D,flags", [(1, 1, 0, 3), (4, 2, 1, 3), (8, 4, 2, 3), (8, 4, 2, 0), (6, 3, 2, 1)])
def test_greedy_equals_sequential_argmax(orc, L, K, D, flags):
    V, N, salt = 6, 24, 3
    cfg = orc.gen_cfg(L=L, V=V, K=K, D=D, flags=flags, n_prompt=len(PROMPT), n_gen=N, toy_salt=salt, top_k=1)
    out, steps, _ = orc.generate(cfg, PROMPT)
    ctx = list(PROMPT)
    ref = []
    for _ in range(N):
        l = orc.toy_logits(np.array(ctx, np.int32), V, salt)
        x = int(np.lexsort((np.arange(V), -l.astype(np.float64)))[0])
        ref.append(x)
        ctx.append(x)
    assert out[:N].tolist() == ref
