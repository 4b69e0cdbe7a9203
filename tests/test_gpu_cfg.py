"""Classifier-free guidance on the GPU (Sec. 5.1 samples with guidance
weight 3: l = l_u + w (l_c - l_u)), through the C ABI. A guided context runs
the text-prompt stream and the unconditional stream in one window forward
(rows [0, L) and [32, 32 + L)), each on its own cache and positions.
- the guided window logits against the oracle: two plain oracle forwards
  (one per prompt, each stream at its own positions) and the oracle's
  combine; prompts of unequal lengths on both sides;
- an unconditional prompt equal to the text prompt gives the unguided
  logits and tokens;
- greedy decoding of a guided window equals guided one-slot decoding (the
  Jacobi fixed point of the guided model);
- the law of the first guided token matches the oracle's guided softmax
  (chi-square over seeded GPU runs);
- mean committed tokens per step of guided GPU and oracle generations.
"""
import numpy as np
import pytest
import torch

from model_util import causal, make_engine, placeholders, setup, weights_device, weights_numpy
from synth_inputs import model_config, model_weights, prompt_tokens

pytestmark = pytest.mark.gpu

# Each stream's logits are held to 3e-2 (the unguided window forward bound);
# the guided logits u + w (c - u) then carry at most (|1 - w| + |w|) times it.
STREAM_TOL = 3e-2


def guided_tol(w):
    return (abs(1.0 - w) + abs(w)) * STREAM_TOL


def oracle_stream_window(orc, cfg, w_np, prompt, spine):
    """One stream's first-window logits: prefill prompt[:-1], then the
    window (prompt[-1], spine...) at positions n .. n + L - 1."""
    m = orc.Model(cfg, w_np, max_seq=cfg["max_seq"])
    n = len(prompt) - 1
    for s0 in range(0, n, 64):
        M = min(64, n - s0)
        m.forward(s0, list(prompt[s0:s0 + M]), list(range(s0, s0 + M)), causal(M), logits=False)
    L = cfg["L"]
    toks = [int(prompt[-1])] + list(spine[:L - 1])
    out = m.forward(n, toks, [n + i for i in range(L)], causal(L))
    m.close()
    return out


def guided_engine(cfg, wd, prompt, uncond, seed):
    eng = make_engine(cfg, wd)
    eng.prefill_cfg(prompt.cuda(), uncond.cuda(), seed)
    return eng


FWD_CASES = [
    ("tiny", {"L": 16}, 9),    # unconditional prompt longer than the text prompt
    ("tiny", {"L": 32}, 5),    # shorter; a full 32-row stream
    ("7b", {"n_layers": 2, "n_prompt": 40, "L": 32}, 70),  # more than one prefill window
    # 128-dim heads over long caches (many key chunks in both streams)
    ("tiny", {"n_layers": 1, "d_model": 512, "n_heads": 4, "n_kv_heads": 2, "head_dim": 128, "ffn_dim": 1024,
              "n_prompt": 700, "L": 32, "weights_f32": False}, 1100),
]


@pytest.mark.parametrize("name,over,n_u", FWD_CASES, ids=[f"{n}-{i}" for i, (n, _, _) in enumerate(FWD_CASES)])
@pytest.mark.parametrize("w", [3.0, -0.5])
def test_guided_window_forward_matches_oracle(orc, name, over, n_u, w):
    cfg = model_config(name, cfg_w=w, **over)
    cfg["max_seq"] = max(cfg["max_seq"], n_u + 2 * cfg["L"] + 8)
    wt, prompt = setup(cfg, wseed=41, pseed=42, device="cuda")
    uncond = prompt_tokens(dict(cfg, n_prompt=n_u), 43)
    seed = 6
    print(f"case {name} {over} n_u={n_u} w={w}", flush=True)
    eng = guided_engine(cfg, weights_device(wt), prompt, uncond, seed)
    got_t = torch.empty(cfg["L"], cfg["V"], dtype=torch.float32, device="cuda")
    eng.forward_window(got_t)
    torch.cuda.synchronize()
    got = got_t.cpu().numpy()
    eng.close()
    w_np = weights_numpy(wt)
    spine = placeholders(orc, cfg, seed)
    lc = oracle_stream_window(orc, cfg, w_np, prompt.numpy(), spine)
    lu = oracle_stream_window(orc, cfg, w_np, uncond.numpy(), spine)
    ref = orc.cfg_combine(lc, lu, w)
    err = np.abs(got - ref).max()
    # a window that mixed up the streams, caches or positions would be far off
    wrong = min(np.abs(got - lc).max(), np.abs(got - lu).max())
    print(f"{name} {over} w={w}: max |guided logit error| = {err:.3e} (tol {guided_tol(w):.3e}); "
          f"distance to either stream alone {wrong:.3f}", flush=True)
    assert np.isfinite(got).all()
    assert err <= guided_tol(w), err
    assert wrong > 3 * guided_tol(w)


def generate(eng, cfg, *, seed, n_gen, top_k, T=1.0, max_steps=10_000):
    meta = torch.zeros(8, dtype=torch.int32, device="cuda")
    tok = torch.zeros(cfg["L"], dtype=torch.int32, device="cuda")
    out, ncs, ns = [], [], []
    step = 0
    while len(out) < n_gen and step < max_steps:
        eng.step(T, top_k, seed, step, out_meta=meta, out_tok=tok)
        m = meta.cpu().numpy()
        t = tok.cpu().numpy()
        n_c = int(m[0])
        assert 1 <= n_c <= cfg["L"], m
        out.extend(t[:n_c].tolist())
        ncs.append(n_c)
        ns.append(int(m[7]))
        step += 1
    return out[:n_gen], ncs, ns


def test_identical_prompts_equal_unguided():
    cfg = model_config("tiny", n_gen=96)
    wt, prompt = setup(cfg, wseed=51, pseed=52)
    wd = weights_device(wt)
    plain = make_engine(cfg, wd)
    plain.prefill(prompt.cuda(), 4)
    l0 = torch.empty(cfg["L"], cfg["V"], dtype=torch.float32, device="cuda")
    plain.forward_window(l0)
    toks0, _, _ = generate(plain, cfg, seed=4, n_gen=96, top_k=1)
    plain.close()
    gcfg = dict(cfg, cfg_w=3.0)
    g = guided_engine(gcfg, wd, prompt, prompt, 4)
    l1 = torch.empty_like(l0)
    g.forward_window(l1)
    toks1, _, ns = generate(g, gcfg, seed=4, n_gen=96, top_k=1)
    g.close()
    err = (l0 - l1).abs().max().item()
    print(f"identical prompts: max |guided - unguided| = {err:.3e}")
    assert err <= 1e-4
    assert toks0 == toks1


@pytest.mark.parametrize("n_u,K,D,flags", [(24, 4, 3, 3), (9, 2, 2, 1), (16, 1, 0, 0)])
def test_guided_greedy_window_equals_guided_autoregressive(n_u, K, D, flags):
    base = model_config("tiny", K=K, D=D, flags=flags, L=16, cfg_w=3.0)
    base["max_seq"] = max(base["max_seq"], n_u + base["n_gen"] + 2 * base["L"] + 8)
    wt, prompt = setup(base, wseed=61, pseed=62)
    uncond = prompt_tokens(dict(base, n_prompt=n_u), 63)
    wd = weights_device(wt)
    eng = guided_engine(base, wd, prompt, uncond, 1)
    win, ncs, ns = generate(eng, base, seed=1, n_gen=96, top_k=1)
    eng.close()
    ar_cfg = dict(base, L=1, K=1, D=0)
    eng = guided_engine(ar_cfg, wd, prompt, uncond, 1)
    ar, ar_ncs, _ = generate(eng, ar_cfg, seed=1, n_gen=96, top_k=1)
    eng.close()
    # the text stream's cache grows by the committed count
    assert ns == list(np.cumsum(ncs) + base["n_prompt"] - 1)
    assert set(ar_ncs) == {1}
    assert win == ar
    assert np.mean(ncs) > 1.0


def pooled_chisquare(counts, expected):
    """Chi-square with cells of expected count < 5 pooled into one."""
    from scipy import stats
    small = expected < 5
    c = np.append(counts[~small], counts[small].sum())
    e = np.append(expected[~small], expected[small].sum())
    if e[-1] == 0:
        c, e = c[:-1], e[:-1]
    return stats.chisquare(c, e)


def test_first_guided_token_law(orc):
    cfg = model_config("tiny", n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, ffn_dim=128,
                       vocab_size=32, V=32, L=4, K=2, D=1, n_prompt=3, n_gen=1, cfg_w=3.0)
    wt = model_weights(cfg, 71, std=0.08)
    prompt = torch.tensor([1, 5, 2], dtype=torch.int32)
    uncond = torch.tensor([6, 0, 3, 7, 4], dtype=torch.int32)
    w_np = weights_numpy(wt)
    m = orc.Model(cfg, w_np, max_seq=cfg["max_seq"] + 16)

    def last_logits(p):
        n = len(p) - 1
        m.forward(0, list(p[:n]), list(range(n)), causal(n), logits=False)
        return m.forward(n, [int(p[-1])], [n], [1])[0]
    lc = last_logits(prompt.numpy())
    lu = last_logits(uncond.numpy())
    m.close()
    l = orc.cfg_combine(lc, lu, 3.0).astype(np.float64)
    law = np.exp(l - l.max())
    law /= law.sum()
    eng = make_engine(cfg, weights_device(wt))
    runs = 3000
    counts = np.zeros(cfg["V"])
    meta = torch.zeros(8, dtype=torch.int32, device="cuda")
    tok = torch.zeros(cfg["L"], dtype=torch.int32, device="cuda")
    pc, uc = prompt.cuda(), uncond.cuda()
    for r in range(runs):
        eng.prefill_cfg(pc, uc, 20_000 + r)
        eng.step(1.0, 0, 20_000 + r, 0, out_meta=meta, out_tok=tok)
        counts[int(tok[0].item())] += 1
    eng.close()
    chi2, pval = pooled_chisquare(counts, law * runs)
    print(f"law {np.round(law, 3)}\ncounts {np.round(counts / runs, 3)} p={pval:.3g}")
    assert pval > 1e-4
    # guidance changed the law: the text-prompt law alone is rejected
    lc64 = lc.astype(np.float64)
    law_c = np.exp(lc64 - lc64.max())
    law_c /= law_c.sum()
    assert pooled_chisquare(counts, law_c * runs)[1] < 1e-6


def test_guided_acceptance_statistics_match_oracle(orc):
    cfg = model_config("tiny", n_gen=128, cfg_w=3.0)
    wt, prompt = setup(cfg, wseed=81, pseed=82)
    uncond = prompt_tokens(dict(cfg, n_prompt=11), 83)
    eng = make_engine(cfg, weights_device(wt))
    gpu = []
    for s in range(12):
        eng.prefill_cfg(prompt.cuda(), uncond.cuda(), 300 + s)
        _, ncs, _ = generate(eng, cfg, seed=300 + s, n_gen=128, top_k=0)
        gpu += ncs
    eng.close()
    m = orc.Model(cfg, weights_numpy(wt), max_seq=cfg["max_seq"])
    ocfg = orc.ModelCfg(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"],
                        cfg["ffn_dim"], cfg["vocab_size"], cfg["vis_lo"], cfg["V"], cfg["max_seq"], 1e-5, 1e4)
    orc_nc = []
    for s in range(12):
        g = orc.gen_cfg(L=cfg["L"], V=cfg["V"], K=cfg["K"], D=cfg["D"], top_k=0, seed=400 + s,
                        n_prompt=cfg["n_prompt"], n_gen=128, mcfg=ocfg, weights=m.w, cfg_w=3.0,
                        uncond=uncond.numpy())
        _, steps, hist = orc.generate(g, prompt.numpy().astype(np.int32))
        orc_nc += sum(([i] * int(c) for i, c in enumerate(hist)), [])
    m.close()
    a, b = np.array(gpu, float), np.array(orc_nc, float)
    se = np.sqrt(a.var() / a.size + b.var() / b.size)
    print(f"guided: mean n_c gpu {a.mean():.3f} ({a.size} steps) oracle {b.mean():.3f} ({b.size} steps) se {se:.3f}")
    assert abs(a.mean() - b.mean()) < 4 * se + 0.02
