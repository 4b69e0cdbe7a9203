"""Oracle-side helpers shared by the tests, the smoke check and the
benchmark's CPU-baseline leg: bf16 weights as the oracle reads them, the
placeholder window of a fresh generation, prefill of the oracle's cache and
its first window.

TEST INFRASTRUCTURE (like the rest of this package): the product path never
imports it.
"""
import numpy as np

NAMES = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"]


def weights_numpy(w):
    """torch weights -> numpy for the oracle (bf16 as raw uint16 words)."""
    import torch

    def cv(t):
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.float().numpy()
    return dict(embed=cv(w["embed"]), final_norm=cv(w["final_norm"]), lm_head=cv(w["lm_head"]),
                layers=[{k: cv(v) for k, v in l.items()} for l in w["layers"]])


def causal(M):
    return [(1 << (a + 1)) - 1 for a in range(M)]


def forced(cfg, g):
    W = cfg.get("row_len", 0)
    return W > 0 and g >= 0 and g % (W + 1) == W


def placeholders(orc, cfg, seed):
    """The first window's drafts: uniform over the support from the
    placeholder stream (tag 6, trial 0, step word 0xFFFFFFFF), row ends forced."""
    out = []
    for i in range(cfg["L"]):
        if forced(cfg, i):
            out.append(cfg["eol_id"])
        else:
            b = orc.bits(seed, orc.TAG_INIT, 0, i, 0, 0xFFFFFFFF, 0)
            out.append(cfg["vis_lo"] + ((b * cfg["V"]) >> 32))
    return out


def oracle_model(orc, cfg, w_np, max_seq=None):
    return orc.Model(cfg, w_np, max_seq=max_seq or cfg["max_seq"])


def oracle_prefill(m, prompt, start=0):
    """Caches prompt[start .. len-1) (the last token is the pending one) in
    64-slot causal windows; returns the cached row count."""
    n = len(prompt) - 1
    for s0 in range(start, n, 64):
        M = min(64, n - s0)
        m.forward(s0, prompt[s0:s0 + M], list(range(s0, s0 + M)), causal(M), logits=False)
    return n


def oracle_first_window(orc, cfg, w_np, prompt, seed):
    m = oracle_model(orc, cfg, w_np)
    n = oracle_prefill(m, prompt)
    L = cfg["L"]
    spine = placeholders(orc, cfg, seed)
    toks = [int(prompt[-1])] + spine[:L - 1]
    logits = m.forward(n, toks, [n + i for i in range(L)], causal(L))
    m.close()
    return logits
