"""Helpers shared by the model-level GPU tests: weight conversion for the
oracle, the oracle's first window after prefill, and engine construction."""
import numpy as np
import torch

from synth_inputs import model_weights, prompt_tokens

NAMES = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"]


def weights_numpy(w):
    """torch weights -> numpy for the oracle (bf16 as raw uint16 words)."""
    def cv(t):
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.float().numpy()
    return dict(embed=cv(w["embed"]), final_norm=cv(w["final_norm"]), lm_head=cv(w["lm_head"]),
                layers=[{k: cv(v) for k, v in l.items()} for l in w["layers"]])


def weights_device(w):
    return dict(embed=w["embed"].cuda(), final_norm=w["final_norm"].cuda(), lm_head=w["lm_head"].cuda(),
                layers=[{k: v.cuda() for k, v in l.items()} for l in w["layers"]])


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


def oracle_model(orc, cfg, w_np):
    return orc.Model(cfg, w_np, max_seq=cfg["max_seq"])


def oracle_prefill(m, prompt):
    n = len(prompt) - 1
    for s0 in range(0, n, 64):
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


def make_engine(cfg, w_dev):
    from paper_2603_18599_amd.sjd import Engine
    return Engine(cfg, w_dev)


def setup(name_cfg, wseed=1, pseed=2, device="cpu"):
    """Seeded weights and prompt; generated on `device` (the GPU is much
    faster for the large shapes) and returned on the CPU."""
    w = model_weights(name_cfg, wseed, device=device)
    if device != "cpu":
        w = dict(embed=w["embed"].cpu(), final_norm=w["final_norm"].cpu(), lm_head=w["lm_head"].cpu(),
                 layers=[{k: v.cpu() for k, v in l.items()} for l in w["layers"]])
    prompt = prompt_tokens(name_cfg, pseed)
    return w, prompt
