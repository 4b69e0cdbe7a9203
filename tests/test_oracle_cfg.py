"""Pins for the oracle's classifier-free guidance (the paper samples with a
CFG weight of 3, Sec. 5.1; l = l_u + w (l_c - l_u), the standard
logit-space guidance):
- the combine's special cases (w = 0 gives the unconditional logits, w = 1
  the conditional ones, identical inputs are a fixed point for any w, and it
  is affine in w);
- a guided generation whose unconditional prompt equals the text prompt is
  token for token the unguided generation (the second stream, its cache,
  positions and pending token are then invisible);
- the law of the first guided token equals the softmax of the guided logits,
  these computed here from two plain oracle forwards (one per prompt) and
  numpy, by a chi-square test over seeded generations. A guided step that
  used the wrong stream, positions or pending token would change the law.
"""
import numpy as np
import pytest
from scipy import stats

from model_util import weights_numpy
from synth_inputs import model_config, model_weights


def test_combine_special_cases(orc):
    rng = np.random.default_rng(3)
    lc = rng.normal(0, 3, 4096).astype(np.float32)
    lu = rng.normal(0, 3, 4096).astype(np.float32)
    assert np.array_equal(orc.cfg_combine(lc, lu, 0.0), lu)
    assert np.abs(orc.cfg_combine(lc, lu, 1.0) - lc).max() <= 4 * np.finfo(np.float32).eps * np.abs(lc).max()
    for w in (0.0, 1.0, 3.0, -2.5):
        assert np.array_equal(orc.cfg_combine(lc, lc, w), lc)
    g2, g3 = orc.cfg_combine(lc, lu, 2.0).astype(np.float64), orc.cfg_combine(lc, lu, 3.0).astype(np.float64)
    assert np.allclose(g3 - g2, lc.astype(np.float64) - lu, atol=1e-5)  # affine in w


def micro_cfg(**over):
    c = model_config("tiny", n_layers=1, d_model=64, n_heads=2, n_kv_heads=2, head_dim=32, ffn_dim=128,
                     vocab_size=8, V=8, L=4, K=2, D=1, n_prompt=3, n_gen=4, **over)
    return c


def oracle_model(orc, cfg, seed, std):
    w = model_weights(cfg, seed, std=std)
    m = orc.Model(cfg, weights_numpy(w), max_seq=cfg["max_seq"] + 16)
    ocfg = orc.ModelCfg(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"],
                        cfg["ffn_dim"], cfg["vocab_size"], cfg["vis_lo"], cfg["V"], cfg["max_seq"] + 16, 1e-5, 1e4)
    return m, ocfg


def test_cfg_identical_prompts_is_unguided(orc):
    cfg = model_config("tiny", n_gen=48)
    m, ocfg = oracle_model(orc, cfg, 5, 0.02)
    prompt = np.arange(3, 3 + cfg["n_prompt"], dtype=np.int32) % cfg["V"]
    for seed in (1, 2):
        g0 = orc.gen_cfg(L=cfg["L"], V=cfg["V"], K=cfg["K"], D=cfg["D"], seed=seed, n_prompt=len(prompt),
                         n_gen=48, mcfg=ocfg, weights=m.w)
        g1 = orc.gen_cfg(L=cfg["L"], V=cfg["V"], K=cfg["K"], D=cfg["D"], seed=seed, n_prompt=len(prompt),
                         n_gen=48, mcfg=ocfg, weights=m.w, cfg_w=3.0, uncond=prompt)
        t0, s0, _ = orc.generate(g0, prompt)
        t1, s1, _ = orc.generate(g1, prompt)
        assert np.array_equal(t0, t1) and s0 == s1
    m.close()


def guided_first_token_law(orc, m, prompt, uncond, w):
    def last_logits(p):
        n = len(p) - 1
        for s in range(0, n, 64):  # prefill
            k = min(64, n - s)
            m.forward(s, list(p[s:s + k]), list(range(s, s + k)),
                      [(1 << (a + 1)) - 1 for a in range(k)], logits=False)
        return m.forward(n, [int(p[-1])], [n], [1])[0]
    lc = last_logits(prompt)
    lu = last_logits(uncond)  # rows of the first prompt are overwritten: same layout, new content
    l = orc.cfg_combine(lc, lu, w).astype(np.float64)
    p = np.exp(l - l.max())
    return p / p.sum()


@pytest.mark.parametrize("w", [3.0, -1.0])
def test_cfg_first_token_law(orc, w):
    cfg = micro_cfg()
    m, ocfg = oracle_model(orc, cfg, 7, 0.08)
    prompt = np.array([1, 5, 2], np.int32)
    uncond = np.array([6, 0, 3, 7, 4], np.int32)
    law = guided_first_token_law(orc, m, prompt, uncond, w)
    assert law.min() > 1e-3
    runs = 3000
    counts = np.zeros(cfg["V"])
    for r in range(runs):
        g = orc.gen_cfg(L=cfg["L"], V=cfg["V"], K=cfg["K"], D=cfg["D"], seed=10_000 + r, n_prompt=len(prompt),
                        n_gen=1, mcfg=ocfg, weights=m.w, cfg_w=w, uncond=uncond)
        toks, _, _ = orc.generate(g, prompt)
        counts[toks[0]] += 1
    m.close()
    chi2, pval = stats.chisquare(counts, law * runs)
    print(f"w={w}: law {np.round(law, 3)} counts {counts / runs} p={pval:.3g}")
    assert pval > 1e-4
    # and guidance mattered: the unguided law differs
    assert np.abs(law - guided_first_token_law(orc, oracle_model(orc, cfg, 7, 0.08)[0], prompt, uncond, 1.0)).max() > 0.02
