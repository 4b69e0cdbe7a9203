"""Pin for the oracle's KV bookkeeping inside a transformer generation (the
"KV cache update & backtracking" phase of Tab. 4 in Appendix B; the drafted
siblings of Sec. 4.1).

Causality fixes the cache: after any sequence of steps, the keys and values
cached for positions [0, n) are those of a plain prefill of the prompt plus
the committed tokens (cache = recompute). A step that accepts a drafted
sibling commits it from a sibling slot, whose key/value row must move into
the committed prefix; a wrong source or destination row leaves a stale or
rejected token's row behind, which this comparison sees. The generations
below accept siblings at several steps (checked), with and without
classifier-free guidance (two caches).
"""
import numpy as np
import pytest

import test_oracle_forward as tf

PROMPT = np.array([1, 5, 9, 20, 33, 12], np.int32)
UNCOND = np.array([3, 44, 7], np.int32)


def _prefill_rows(orc, cfg, wt, tokens, max_seq):
    """A fresh cache holding tokens[0 .. len) (64-slot causal windows)."""
    m = orc.Model(cfg, tf.to_numpy(wt), max_seq=max_seq)
    n = len(tokens)
    for s0 in range(0, n, 64):
        M = min(64, n - s0)
        m.forward(s0, tokens[s0:s0 + M], list(range(s0, s0 + M)), [(1 << (a + 1)) - 1 for a in range(M)],
                  logits=False)
    return m


def _max_row_diff(a, b, n_layers, n):
    worst = 0.0
    for l in range(n_layers):
        for r in range(n):
            ka, va = a.kv_row(l, r)
            kb, vb = b.kv_row(l, r)
            worst = max(worst, float(np.abs(ka - kb).max()), float(np.abs(va - vb).max()))
    return worst


@pytest.mark.parametrize("seed,T,L,K,D", [(0, 1.0, 8, 3, 2), (1, 2.0, 8, 3, 2), (2, 1.0, 10, 4, 2)])
def test_cache_equals_recompute_after_sibling_commits(orc, seed, T, L, K, D):
    cfg = dict(tf.CFG)
    wt = tf.make_weights(cfg, 3)
    max_seq = 200
    m = orc.Model(cfg, tf.to_numpy(wt), max_seq=max_seq)
    try:
        g = orc.gen_cfg(L=L, V=cfg["V"], K=K, D=D, top_k=0, T=T, flags=orc.AC | orc.PD, seed=seed,
                        n_prompt=len(PROMPT), n_gen=60, vis_lo=cfg["vis_lo"], mcfg=m.cfg, weights=m.w)
        out, steps, _, sm = orc.generate(g, PROMPT, step_meta=True, model=m)
        assert (sm[:, 5] >= 2).sum() >= 2, "no step accepted a drafted sibling"
        assert int(sm[:, 0].sum()) == len(out)
        n = len(PROMPT) - 1 + len(out)  # cached rows: everything but the pending token
        ref = _prefill_rows(orc, cfg, wt, np.concatenate([PROMPT, out])[:n], max_seq)
        try:
            diff = _max_row_diff(m, ref, cfg["n_layers"], n)
        finally:
            ref.close()
        assert diff <= 1e-9, f"cached rows differ from a recompute by {diff}"
    finally:
        m.close()


def test_guided_caches_equal_recompute_after_sibling_commits(orc):
    cfg = dict(tf.CFG)
    wt = tf.make_weights(cfg, 3)
    max_seq = 200
    m = orc.Model(cfg, tf.to_numpy(wt), max_seq=max_seq)
    mu = orc.Model(cfg, tf.to_numpy(wt), max_seq=max_seq)
    try:
        g = orc.gen_cfg(L=8, V=cfg["V"], K=3, D=2, top_k=0, T=1.0, flags=orc.AC | orc.PD, seed=4,
                        n_prompt=len(PROMPT), n_gen=60, vis_lo=cfg["vis_lo"], mcfg=m.cfg, weights=m.w,
                        cfg_w=3.0, uncond=UNCOND)
        out, steps, _, sm = orc.generate(g, PROMPT, step_meta=True, model=m, model_u=mu)
        assert (sm[:, 5] >= 2).sum() >= 1, "no step accepted a drafted sibling"
        for prompt, cache in ((PROMPT, m), (UNCOND, mu)):
            n = len(prompt) - 1 + len(out)
            ref = _prefill_rows(orc, cfg, wt, np.concatenate([prompt, out])[:n], max_seq)
            try:
                diff = _max_row_diff(cache, ref, cfg["n_layers"], n)
            finally:
                ref.close()
            assert diff <= 1e-9, f"cached rows differ from a recompute by {diff}"
    finally:
        m.close()
        mu.close()
