"""Helpers shared by the model-level GPU tests: engine construction and
device weights; the oracle-side helpers live in oracle/harness.py."""
import torch  # noqa: F401

from oracle.harness import (NAMES, causal, forced, oracle_first_window, oracle_model,  # noqa: F401
                            oracle_prefill, placeholders, weights_numpy)
from synth_inputs import model_weights, prompt_tokens


def weights_device(w):
    return dict(embed=w["embed"].cuda(), final_norm=w["final_norm"].cuda(), lm_head=w["lm_head"].cuda(),
                layers=[{k: v.cuda() for k, v in l.items()} for l in w["layers"]])


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
