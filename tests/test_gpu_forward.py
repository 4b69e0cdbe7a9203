"""GPU window forward (bf16 MFMA path, through the C ABI) against the
oracle's fp64-accumulated forward on the same weights, prompt and window:
logits within 3e-2 max-abs. Shapes: the tiny and mid models, slices (few
layers) of the 7B-shaped and 8B GQA large-vocabulary models at their full
widths (also at the benchmarked cache lengths), the full 32-layer 7B-shaped
and 8B GQA models (the benchmarked models, after a short prompt), and
narrow models with 128-dim heads over caches of 700-2100 rows (the
split-KV attention with many chunks)."""
import numpy as np
import pytest
import torch

from model_util import make_engine, oracle_first_window, setup, weights_device, weights_numpy
from synth_inputs import model_config

pytestmark = pytest.mark.gpu

TOL = 3e-2

CASES = [
    ("tiny", {}),
    ("mid", {"n_layers": 3}),
    ("7b", {"n_layers": 2, "n_prompt": 40}),
    ("8b", {"n_layers": 2, "n_prompt": 24}),
    ("tiny", {"L": 7, "K": 2, "D": 3, "n_prompt": 1}),
    ("mid", {}),
    ("7b", {"n_prompt": 16}),
    ("8b", {"n_prompt": 16}),
    # the benchmarked widths at the benchmarked cache lengths: a 7B slice
    # after 1239 cached rows (ten 128-key chunks per head) and an 8B GQA
    # slice after 4158 (33 chunks per key/value head)
    ("7b", {"n_layers": 2, "n_prompt": 1240}),
    ("8b", {"n_layers": 1, "n_prompt": 4159}),
    # windows of up to 64 slots: two 32-row GEMM tiles, two attention slot
    # halves; prompts longer than one 64-token prefill window
    ("tiny", {"L": 64, "n_prompt": 100}),
    ("7b", {"n_layers": 2, "L": 64, "n_prompt": 70}),
    ("8b", {"n_layers": 2, "L": 48, "n_prompt": 40}),
    # 128-dim heads over long caches: the split-KV attention with many
    # 128-key chunks and their combine (the 7B benchmark step takes 10 chunks
    # per head at 1239 cached rows; prefill windows of 64 rows take two slot
    # halves), on narrow bf16 models so that the oracle's prefill stays quick
    ("tiny", {"n_layers": 1, "d_model": 512, "n_heads": 4, "n_kv_heads": 4, "head_dim": 128, "ffn_dim": 1024,
              "n_prompt": 1271, "L": 32, "weights_f32": False}),
    ("tiny", {"n_layers": 2, "d_model": 512, "n_heads": 4, "n_kv_heads": 2, "head_dim": 128, "ffn_dim": 1024,
              "n_prompt": 700, "weights_f32": False}),
    ("tiny", {"n_layers": 1, "d_model": 256, "n_heads": 2, "n_kv_heads": 2, "head_dim": 128, "ffn_dim": 512,
              "n_prompt": 2100, "L": 64, "weights_f32": False}),
]


@pytest.mark.parametrize("name,over", CASES, ids=[f"{n}-{i}" for i, (n, _) in enumerate(CASES)])
def test_window_forward_matches_oracle(orc, name, over):
    cfg = model_config(name, **over)
    w, prompt = setup(cfg, wseed=11, pseed=12, device="cuda")
    seed = 5
    print(f"case {name} {over}", flush=True)
    eng = make_engine(cfg, weights_device(w))
    eng.prefill(prompt.cuda(), seed)
    logits = torch.empty(cfg["L"], cfg["V"], dtype=torch.float32, device="cuda")
    eng.forward_window(logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    eng.close()
    ref = oracle_first_window(orc, cfg, weights_numpy(w), prompt.numpy().astype(np.int32), seed)
    err = np.abs(got - ref).max()
    print(f"{name} {over}: max |logit error| = {err:.3e}, logit std = {ref.std():.3f}", flush=True)
    assert np.isfinite(got).all()
    assert err <= TOL, err


@pytest.mark.parametrize("plan", ["1,1,1,1", "7,3,5,11", "32,32,2,32", "7:8,3,5:8,11:8", "1:8,32:8,2:8,32:8"])
def test_window_forward_under_pinned_split_plans(orc, monkeypatch, plan):
    """The GEMM plan is chosen at init (timed, or pinned by SJD_SPLITS);
    the forward must match the oracle under any plan, including uneven
    splits of the K range, the extremes (no split, more splits than k-steps)
    and 8 column blocks per workgroup (":8")."""
    cfg = model_config("mid", n_layers=2)
    w, prompt = setup(cfg, wseed=13, pseed=14, device="cuda")
    monkeypatch.setenv("SJD_SPLITS", plan)
    eng = make_engine(cfg, weights_device(w))
    entries = [e.split(":") for e in plan.split(",")]
    assert eng.plan()[:4] == [int(e[0]) for e in entries]
    assert eng.plan()[5:9] == [int(e[1]) if len(e) > 1 else 4 for e in entries]
    eng.prefill(prompt.cuda(), 5)
    logits = torch.empty(cfg["L"], cfg["V"], dtype=torch.float32, device="cuda")
    eng.forward_window(logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    eng.close()
    ref = oracle_first_window(orc, cfg, weights_numpy(w), prompt.numpy().astype(np.int32), 5)
    err = np.abs(got - ref).max()
    print(f"plan {plan}: max |logit error| = {err:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert err <= TOL, err


@pytest.mark.parametrize("plan", ["3:8,2:8,2:8,3:8", "1:8,1,3:8,1:8"])
def test_window_forward_wide_groups_with_idle_waves(orc, monkeypatch, plan):
    """8 column blocks per workgroup on a model whose projections are not
    whole groups of 8 blocks (QKV 18 blocks, O and down 6, gate|up 24):
    the waves past the last block stage their share of the activation
    tile, take part in every barrier and store nothing."""
    cfg = model_config("tiny", d_model=192, n_heads=3, n_kv_heads=3, head_dim=64, ffn_dim=384)
    w, prompt = setup(cfg, wseed=15, pseed=16, device="cuda")
    monkeypatch.setenv("SJD_SPLITS", plan)
    eng = make_engine(cfg, weights_device(w))
    eng.prefill(prompt.cuda(), 5)
    logits = torch.empty(cfg["L"], cfg["V"], dtype=torch.float32, device="cuda")
    eng.forward_window(logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    eng.close()
    ref = oracle_first_window(orc, cfg, weights_numpy(w), prompt.numpy().astype(np.int32), 5)
    err = np.abs(got - ref).max()
    print(f"plan {plan}: max |logit error| = {err:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert err <= TOL, err


@pytest.mark.parametrize("plan", ["5:6,8,4,8", "5,8,4", "0,8,4,8", "33,8,4,8", "5,8,4,8,", "5:,8,4,8", "a,8,4,8"])
def test_malformed_plan_pins_are_rejected(monkeypatch, plan):
    """SJD_SPLITS takes four entries S or S:blocks (1 <= S <= 32, blocks 4
    or 8); anything else fails sjd_init with SJD_EINVAL before any launch."""
    from paper_2603_18599_amd.sjd import SjdError
    cfg = model_config("tiny", n_layers=1)
    w, _ = setup(cfg, wseed=17, pseed=18)
    monkeypatch.setenv("SJD_SPLITS", plan)
    with pytest.raises(SjdError) as e:
        make_engine(cfg, weights_device(w))
    assert e.value.code == -1


def test_window_forward_query_head_split_is_bitwise_neutral(orc, monkeypatch):
    """Grouped-query attention splits a key / value head's query heads over
    SJD_QPARTS workgroups (default one per query head): 1, 2 and 4 query
    heads per workgroup (4 query heads per key / value head, 128-dim heads,
    a cache of 700 rows: many 128-key chunks) give bitwise identical logits,
    which match the oracle; a part count that does not divide the group
    fails sjd_init."""
    cfg = model_config("tiny", n_layers=2, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=1024,
                       n_prompt=700, weights_f32=False)
    w, prompt = setup(cfg, wseed=21, pseed=22, device="cuda")
    outs = {}
    for qp in ("1", "2", "4", ""):
        monkeypatch.setenv("SJD_QPARTS", qp)
        eng = make_engine(cfg, weights_device(w))
        eng.prefill(prompt.cuda(), 5)
        logits = torch.empty(cfg["L"], cfg["V"], dtype=torch.float32, device="cuda")
        eng.forward_window(logits)
        torch.cuda.synchronize()
        outs[qp] = logits.cpu().numpy()
        eng.close()
    for qp in ("2", "4", ""):
        assert np.array_equal(outs[qp], outs["1"]), qp
    ref = oracle_first_window(orc, cfg, weights_numpy(w), prompt.numpy().astype(np.int32), 5)
    err = np.abs(outs[""] - ref).max()
    print(f"query-head split: max |logit error| = {err:.3e}", flush=True)
    assert err <= TOL, err
    from paper_2603_18599_amd.sjd import SjdError
    monkeypatch.setenv("SJD_QPARTS", "3")
    with pytest.raises(SjdError) as e:
        make_engine(cfg, weights_device(w))
    assert e.value.code == -1
