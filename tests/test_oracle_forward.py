"""Pins for the oracle's window forward (ParallelForward of Alg. 1).

- against an independent torch CPU implementation built from library
  primitives (matmul, softmax, silu, scaled-dot-product attention);
- invariants fixed by the mathematics rather than by a formula:
  * rotary embeddings make attention depend on relative positions only, so a
    common position shift leaves every logit unchanged;
  * evaluating a prefix into the cache and then a window equals evaluating
    everything at once (cache = recompute);
  * a slot's output does not depend on slots it cannot see (causality/tree);
  * a sibling slot equals the chain forward with that token substituted;
  * grouped-query attention with duplicated key/value heads equals
    multi-head attention.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

CFG = dict(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96, vocab_size=50,
           vis_lo=10, V=30, rms_eps=1e-5, rope_theta=10000.0)


def make_weights(cfg, seed, as_bf16=True, gains=True):
    g = torch.Generator().manual_seed(seed)
    d, H, Hkv, hd, Fd, Vv = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim",
                                                "vocab_size"))

    def w(*shape, std=0.02):
        t = torch.randn(*shape, generator=g) * std
        return t.to(torch.bfloat16).float() if as_bf16 else t

    def gain(n):
        t = (1.0 + 0.1 * torch.randn(n, generator=g)) if gains else torch.ones(n)
        return t.to(torch.bfloat16).float() if as_bf16 else t

    layers = []
    for _ in range(cfg["n_layers"]):
        layers.append(dict(attn_norm=gain(d), wq=w(H * hd, d, std=0.2), wk=w(Hkv * hd, d, std=0.2),
                           wv=w(Hkv * hd, d, std=0.2), wo=w(d, H * hd, std=0.2), ffn_norm=gain(d),
                           wg=w(Fd, d, std=0.2), wu=w(Fd, d, std=0.2), wd=w(d, Fd, std=0.2)))
    return dict(embed=w(Vv, d, std=1.0), layers=layers, final_norm=gain(d), lm_head=w(Vv, d, std=0.2))


def to_numpy(wt):
    def cv(t):
        return t.numpy().astype(np.float32)
    return dict(embed=cv(wt["embed"]), final_norm=cv(wt["final_norm"]), lm_head=cv(wt["lm_head"]),
                layers=[{k: cv(v) for k, v in l.items()} for l in wt["layers"]])


def torch_reference(cfg, wt, toks, pos, anc):
    """All slots at once (no cache): slot a attends to slot b iff bit b of anc[a]."""
    d, H, Hkv, hd = cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    M = len(toks)
    dt = torch.float64
    x = wt["embed"][torch.tensor(toks)].to(dt)
    posd = torch.tensor(pos, dtype=dt)
    inv = cfg["rope_theta"] ** (-torch.arange(0, hd // 2, dtype=dt) * 2 / hd)
    ang = posd[:, None] * inv[None, :]
    cos, sin = torch.cos(ang), torch.sin(ang)
    mask = torch.tensor([[(anc[a] >> b) & 1 for b in range(M)] for a in range(M)], dtype=torch.bool)

    def rms(v, gvec):
        return v * torch.rsqrt((v * v).mean(-1, keepdim=True) + cfg["rms_eps"]) * gvec.to(dt)

    def rope(t):  # [M, heads, hd]
        a, b = t[..., : hd // 2], t[..., hd // 2:]
        c, s = cos[:, None, :], sin[:, None, :]
        return torch.cat([a * c - b * s, a * s + b * c], -1)

    for lw in wt["layers"]:
        h = rms(x, lw["attn_norm"])
        q = rope((h @ lw["wq"].to(dt).T).view(M, H, hd))
        k = rope((h @ lw["wk"].to(dt).T).view(M, Hkv, hd))
        v = (h @ lw["wv"].to(dt).T).view(M, Hkv, hd)
        rep = H // Hkv
        k = k.repeat_interleave(rep, 1)
        v = v.repeat_interleave(rep, 1)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           attn_mask=mask[None])
        x = x + o.transpose(0, 1).reshape(M, H * hd) @ lw["wo"].to(dt).T
        h2 = rms(x, lw["ffn_norm"])
        x = x + (F.silu(h2 @ lw["wg"].to(dt).T) * (h2 @ lw["wu"].to(dt).T)) @ lw["wd"].to(dt).T
    xf = rms(x, wt["final_norm"])
    head = wt["lm_head"][cfg["vis_lo"]: cfg["vis_lo"] + cfg["V"]].to(dt)
    return (xf @ head.T).numpy()


def causal(M):
    return [(1 << (a + 1)) - 1 for a in range(M)]


@pytest.fixture(scope="module")
def model(orc):
    wt = make_weights(CFG, 1)
    m = orc.Model(CFG, to_numpy(wt), max_seq=256)
    yield m, wt
    m.close()


def test_forward_matches_torch_reference(model):
    m, wt = model
    rng = np.random.default_rng(0)
    M = 20
    toks = rng.integers(0, CFG["vocab_size"], M).tolist()
    pos = list(range(M))
    got = m.forward(0, toks, pos, causal(M))
    ref = torch_reference(CFG, wt, toks, pos, causal(M))
    assert np.abs(got - ref).max() < 1e-4 * max(1.0, np.abs(ref).max())


def test_forward_tree_mask_matches_torch(model):
    m, wt = model
    # spine 0..5, then two siblings of depth 1 and one of depth 2
    toks = [3, 7, 11, 13, 17, 19, 23, 29, 31]
    pos = [0, 1, 2, 3, 4, 5, 2, 2, 3]
    anc = causal(6) + [0b11 | (1 << 6), 0b11 | (1 << 7), 0b111 | (1 << 8)]
    got = m.forward(0, toks, pos, anc)
    ref = torch_reference(CFG, wt, toks, pos, anc)
    assert np.abs(got - ref).max() < 1e-4 * max(1.0, np.abs(ref).max())


def test_rope_relative_position_invariance(model):
    m, _ = model
    toks = [5, 9, 14, 22, 31, 40]
    a = m.forward(0, toks, list(range(6)), causal(6))
    b = m.forward(0, toks, [p + 97 for p in range(6)], causal(6))
    assert np.abs(a - b).max() < 1e-5


def test_cache_equals_recompute(model):
    m, _ = model
    rng = np.random.default_rng(1)
    toks = rng.integers(0, CFG["vocab_size"], 40).tolist()
    full = m.forward(0, toks, list(range(40)), causal(40))
    m.forward(0, toks[:17], list(range(17)), causal(17), logits=False)
    m.forward(17, toks[17:29], list(range(17, 29)), causal(12), logits=False)
    tail = m.forward(29, toks[29:], list(range(29, 40)), causal(11))
    assert np.abs(tail - full[29:]).max() < 1e-9


def test_slots_do_not_see_invisible_slots(model):
    m, _ = model
    toks = [4, 8, 15, 16, 23, 42]
    a = m.forward(0, toks, list(range(6)), causal(6))
    toks2 = toks[:3] + [0, 1, 2]
    b = m.forward(0, toks2, list(range(6)), causal(6))
    assert np.abs(a[:3] - b[:3]).max() == 0.0
    assert np.abs(a[3:] - b[3:]).max() > 1e-3


def test_sibling_slot_equals_substituted_chain(model):
    m, _ = model
    prefix = [1, 2, 3, 4]
    m.forward(0, prefix, [0, 1, 2, 3], causal(4), logits=False)
    # window: spine c=9 @4, s0=10 @5, s1=11 @6; sibling of depth 0 (alternative to s0) = 12 @5
    win = m.forward(4, [9, 10, 11, 12], [4, 5, 6, 5], causal(3) + [0b1 | (1 << 3)])
    m.forward(0, prefix, [0, 1, 2, 3], causal(4), logits=False)
    chain = m.forward(4, [9, 12], [4, 5], causal(2))
    assert np.abs(win[3] - chain[1]).max() < 1e-9
    assert np.abs(win[0] - chain[0]).max() < 1e-9


def test_gqa_with_duplicated_heads_equals_mha(orc):
    cfg_g = dict(CFG)
    wt = make_weights(cfg_g, 7)
    cfg_m = dict(CFG, n_kv_heads=CFG["n_heads"])
    rep = CFG["n_heads"] // CFG["n_kv_heads"]
    hd = CFG["head_dim"]
    wm = {k: v for k, v in wt.items()}
    wm["layers"] = []
    for l in wt["layers"]:
        l2 = dict(l)
        for nm in ("wk", "wv"):
            w = l[nm].view(CFG["n_kv_heads"], hd, -1)
            l2[nm] = w.repeat_interleave(rep, 0).reshape(CFG["n_heads"] * hd, -1)
        wm["layers"].append(l2)
    mg = orc.Model(cfg_g, to_numpy(wt), 64)
    mm = orc.Model(cfg_m, to_numpy(wm), 64)
    toks = [1, 5, 9, 33, 2, 7, 12]
    a = mg.forward(0, toks, list(range(7)), causal(7))
    b = mm.forward(0, toks, list(range(7)), causal(7))
    assert np.abs(a - b).max() < 1e-9
    mg.close()
    mm.close()


def test_bf16_words_equal_float_weights(orc):
    wt = make_weights(CFG, 3)
    f32 = to_numpy(wt)

    def bf(a):
        return (a.view(np.uint32) >> 16).astype(np.uint16)
    b16 = dict(embed=bf(f32["embed"]), final_norm=bf(f32["final_norm"]), lm_head=bf(f32["lm_head"]),
               layers=[{k: bf(v) for k, v in l.items()} for l in f32["layers"]])
    ma = orc.Model(CFG, f32, 64)
    mb = orc.Model(CFG, b16, 64)
    toks = [3, 1, 4, 1, 5, 9, 2, 6]
    assert np.array_equal(ma.forward(0, toks, list(range(8)), causal(8)),
                          mb.forward(0, toks, list(range(8)), causal(8)))
    ma.close()
    mb.close()


def test_forward_rejects_bad_arguments(model):
    m, _ = model
    with pytest.raises(ValueError):
        m.forward(0, [1, 2], [0, 1], [1, 0b01])  # slot 1 must see itself
    with pytest.raises(ValueError):
        m.forward(250, [1] * 10, list(range(10)), causal(10))  # past max_seq
    with pytest.raises(ValueError):
        m.forward(0, [CFG["vocab_size"]], [0], [1])
