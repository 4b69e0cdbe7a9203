"""Several images per step (batch = 2 .. 4) on the GPU, through the C ABI:
image b's window occupies rows [32 b, 32 b + L) of one forward (one pass
over the weights), with its own cache, decoder state and prompt; with
guidance (two images), image b's text and unconditional streams occupy rows
[64 b, 64 b + L) and [64 b + 32, 64 b + 32 + L).
- each image's window logits against the oracle's first window of that
  image alone (prompts of different lengths); guided: against the oracle's
  two stream windows of that image and its combine;
- greedy decoding of a batch gives each image the tokens of a one-image
  context on the same prompt (guided: of a guided one-image context), also
  when one image is restarted mid-run while the others continue;
- each image's cache grows by its own committed counts;
- mean committed tokens per step of batched GPU and oracle generations.
"""
import numpy as np
import pytest
import torch

from model_util import make_engine, oracle_first_window, setup, weights_device, weights_numpy
from synth_inputs import model_config, prompt_tokens

pytestmark = pytest.mark.gpu

TOL = 3e-2  # the window forward bound

CASES = [
    # (model, overrides, prompt lengths of images 1.. (image 0: the model's))
    ("tiny", {"L": 16}, (9,)),
    ("tiny", {"L": 32, "K": 2, "D": 2}, (40,)),
    ("7b", {"n_layers": 2, "n_prompt": 40, "L": 32}, (70,)),
    # 128-dim heads over long caches (many key chunks for both images)
    ("tiny", {"n_layers": 1, "d_model": 512, "n_heads": 4, "n_kv_heads": 4, "head_dim": 128, "ffn_dim": 1024,
              "n_prompt": 1200, "L": 32, "weights_f32": False}, (650,)),
    # three and four images (96- and 128-row windows)
    ("tiny", {"L": 16}, (9, 30, 2)),
    ("7b", {"n_layers": 2, "n_prompt": 40, "L": 32}, (70, 11)),
    ("tiny", {"n_layers": 1, "d_model": 512, "n_heads": 8, "n_kv_heads": 2, "head_dim": 128, "ffn_dim": 1024,
              "n_prompt": 900, "L": 32, "weights_f32": False}, (300, 1300, 45)),
]


@pytest.mark.parametrize("name,over,ns", CASES, ids=[f"{n}-{i}" for i, (n, _, _) in enumerate(CASES)])
def test_batched_window_forward_matches_oracle(orc, name, over, ns):
    B = 1 + len(ns)
    cfg = model_config(name, batch=B, **over)
    cfg["max_seq"] = max(cfg["max_seq"], max(ns) + 2 * cfg["L"] + 8)
    wt, p0 = setup(cfg, wseed=91, pseed=92, device="cuda")
    prompts = [p0] + [prompt_tokens(dict(cfg, n_prompt=n), 93 + i) for i, n in enumerate(ns)]
    print(f"case {name} {over} batch {B} prompts {[len(p) for p in prompts]}", flush=True)
    eng = make_engine(cfg, weights_device(wt))
    for b, p in enumerate(prompts):
        eng.prefill_image(b, p.cuda(), 7 + b)
    L, V = cfg["L"], cfg["V"]
    got_t = torch.empty(32 * (B - 1) + L, V, dtype=torch.float32, device="cuda")
    eng.forward_window(got_t)
    torch.cuda.synchronize()
    got = got_t.cpu().numpy()
    eng.close()
    w_np = weights_numpy(wt)
    refs = []
    for b, p in enumerate(prompts):
        ref = oracle_first_window(orc, cfg, w_np, p.numpy().astype(np.int32), 7 + b)
        rows = got[32 * b:32 * b + L]
        err = np.abs(rows - ref).max()
        print(f"{name} {over} image {b}: max |logit error| = {err:.3e}", flush=True)
        assert np.isfinite(rows).all()
        assert err <= TOL, (b, err)
        refs.append(ref)
    # images that read another image's cache or window would be far off
    for b in range(1, B):
        assert np.abs(refs[b] - refs[b - 1]).max() > 10 * TOL


def run_steps(eng, cfg, B, n_steps, *, seed, top_k, T=1.0):
    """n_steps steps; per image the committed tokens, n_c and cached rows."""
    meta = torch.zeros(B, 8, dtype=torch.int32, device="cuda")
    tok = torch.zeros(B, cfg["L"], dtype=torch.int32, device="cuda")
    toks = [[] for _ in range(B)]
    ncs = [[] for _ in range(B)]
    ns = [[] for _ in range(B)]
    for _ in range(n_steps):
        step = run_steps.counter
        run_steps.counter += 1
        eng.step(T, top_k, seed, step, out_meta=meta, out_tok=tok)
        m = meta.cpu().numpy()
        t = tok.cpu().numpy()
        for b in range(B):
            n_c = int(m[b, 0])
            assert 1 <= n_c <= cfg["L"], m
            toks[b].extend(t[b, :n_c].tolist())
            ncs[b].append(n_c)
            ns[b].append(int(m[b, 7]))
    return toks, ncs, ns


run_steps.counter = 0


def single_greedy(cfg, wd, prompt, n_gen):
    c1 = dict(cfg, batch=1)
    eng = make_engine(c1, wd)
    eng.prefill(prompt.cuda(), 1)
    out = []
    while len(out) < n_gen:
        toks, _, _ = run_steps(eng, c1, 1, 1, seed=1, top_k=1)
        out.extend(toks[0])
    eng.close()
    return out[:n_gen]


@pytest.mark.parametrize("K,D,flags,L,B", [(4, 3, 3, 16, 2), (2, 2, 1, 32, 2), (1, 0, 0, 8, 2), (4, 3, 3, 16, 4),
                                           (2, 2, 1, 32, 3)])
def test_batched_greedy_equals_single_image(K, D, flags, L, B):
    cfg = model_config("tiny", K=K, D=D, flags=flags, L=L, batch=B, n_gen=160)
    cfg["max_seq"] = 1024  # 16 steps of up to L tokens
    wt, p0 = setup(cfg, wseed=95, pseed=96)
    prompts = [p0] + [prompt_tokens(dict(cfg, n_prompt=n), 97 + i) for i, n in enumerate((23, 4, 31)[:B - 1])]
    p_new = prompt_tokens(dict(cfg, n_prompt=5), 98)
    wd = weights_device(wt)
    eng = make_engine(cfg, wd)
    for b, p in enumerate(prompts):
        eng.prefill_image(b, p.cuda(), 1 + b)
    t_a, nc_a, ns_a = run_steps(eng, cfg, B, 6, seed=1, top_k=1)
    # restart the last image with a new prompt; the others continue
    eng.prefill_image(B - 1, p_new.cuda(), 3)
    t_b, nc_b, ns_b = run_steps(eng, cfg, B, 10, seed=1, top_k=1)
    eng.close()
    # cache rows grow by each image's own committed counts
    for b, p in enumerate(prompts):
        assert ns_a[b] == list(np.cumsum(nc_a[b]) + len(p) - 1)
    assert ns_b[B - 1] == list(np.cumsum(nc_b[B - 1]) + len(p_new) - 1)
    for b, p in enumerate(prompts[:B - 1]):
        img = t_a[b] + t_b[b]
        assert img == single_greedy(cfg, wd, p, len(img)), b
    assert t_a[B - 1] == single_greedy(cfg, wd, prompts[B - 1], len(t_a[B - 1]))
    assert t_b[B - 1] == single_greedy(cfg, wd, p_new, len(t_b[B - 1]))
    assert np.mean(nc_a[0] + nc_b[0]) > 1.0


GUIDED_CASES = [
    ("tiny", {"L": 16}, (16, 9), (5, 30)),   # (model, overrides, text prompt lengths, unconditional lengths)
    ("7b", {"n_layers": 2, "L": 32}, (40, 70), (12, 71)),
    ("tiny", {"n_layers": 1, "d_model": 512, "n_heads": 4, "n_kv_heads": 2, "head_dim": 128, "ffn_dim": 1024,
              "L": 32, "weights_f32": False}, (700, 300), (1100, 20)),
]


@pytest.mark.parametrize("name,over,n_p,n_u", GUIDED_CASES, ids=[f"{n}-{i}" for i, (n, *_) in enumerate(GUIDED_CASES)])
def test_guided_batch_window_forward_matches_oracle(orc, name, over, n_p, n_u):
    """Two guided images in one forward (four streams): image b's guided rows
    against the oracle's two stream windows of image b and its combine."""
    from test_gpu_cfg import guided_tol, oracle_stream_window
    from model_util import placeholders
    w = 3.0
    cfg = model_config(name, batch=2, cfg_w=w, **over)
    cfg["max_seq"] = max(cfg["max_seq"], max(n_p + n_u) + 2 * cfg["L"] + 8)
    wt, _ = setup(cfg, wseed=111, pseed=112, device="cuda")
    text = [prompt_tokens(dict(cfg, n_prompt=n), 113 + i) for i, n in enumerate(n_p)]
    unc = [prompt_tokens(dict(cfg, n_prompt=n), 123 + i) for i, n in enumerate(n_u)]
    print(f"case {name} {over} text {n_p} uncond {n_u}", flush=True)
    eng = make_engine(cfg, weights_device(wt))
    for b in range(2):
        eng.prefill_cfg(text[b].cuda(), unc[b].cuda(), 9 + b, image=b)
    L, V = cfg["L"], cfg["V"]
    got_t = torch.empty(32 + L, V, dtype=torch.float32, device="cuda")
    eng.forward_window(got_t)
    torch.cuda.synchronize()
    got = got_t.cpu().numpy()
    eng.close()
    w_np = weights_numpy(wt)
    for b in range(2):
        spine = placeholders(orc, cfg, 9 + b)
        lc = oracle_stream_window(orc, cfg, w_np, text[b].numpy(), spine)
        lu = oracle_stream_window(orc, cfg, w_np, unc[b].numpy(), spine)
        ref = orc.cfg_combine(lc, lu, w)
        rows = got[32 * b:32 * b + L]
        err = np.abs(rows - ref).max()
        wrong = min(np.abs(rows - lc).max(), np.abs(rows - lu).max())
        print(f"{name} {over} image {b}: max |guided logit error| = {err:.3e} (tol {guided_tol(w):.3e}); "
              f"distance to either stream alone {wrong:.3f}", flush=True)
        assert np.isfinite(rows).all()
        assert err <= guided_tol(w), (b, err)
        assert wrong > 3 * guided_tol(w)


def test_guided_batch_greedy_equals_guided_single_image():
    """Greedy decoding of two guided images per step gives each image the
    tokens of a guided one-image context with the same prompts, also after
    one image is restarted while the other continues."""
    from test_gpu_cfg import generate
    cfg = model_config("tiny", K=4, D=3, flags=3, L=16, batch=2, cfg_w=3.0, n_gen=160)
    cfg["max_seq"] = 1024
    wt, p0 = setup(cfg, wseed=131, pseed=132)
    p1 = prompt_tokens(dict(cfg, n_prompt=21), 133)
    u0 = prompt_tokens(dict(cfg, n_prompt=7), 134)
    u1 = prompt_tokens(dict(cfg, n_prompt=33), 135)
    p2 = prompt_tokens(dict(cfg, n_prompt=4), 136)
    u2 = prompt_tokens(dict(cfg, n_prompt=12), 137)
    wd = weights_device(wt)
    eng = make_engine(cfg, wd)
    eng.prefill_cfg(p0.cuda(), u0.cuda(), 1, image=0)
    eng.prefill_cfg(p1.cuda(), u1.cuda(), 2, image=1)
    t_a, nc_a, ns_a = run_steps(eng, cfg, 2, 6, seed=1, top_k=1)
    eng.prefill_cfg(p2.cuda(), u2.cuda(), 3, image=1)
    t_b, nc_b, ns_b = run_steps(eng, cfg, 2, 10, seed=1, top_k=1)
    eng.close()
    assert ns_a[0] == list(np.cumsum(nc_a[0]) + len(p0) - 1)
    assert ns_b[1] == list(np.cumsum(nc_b[1]) + len(p2) - 1)

    def single(p, u, n):
        c1 = dict(cfg, batch=1)
        e = make_engine(c1, wd)
        e.prefill_cfg(p.cuda(), u.cuda(), 1)
        out, _, _ = generate(e, c1, seed=1, n_gen=n, top_k=1)
        e.close()
        return out
    img0 = t_a[0] + t_b[0]
    assert img0 == single(p0, u0, len(img0))
    assert t_a[1] == single(p1, u1, len(t_a[1]))
    assert t_b[1] == single(p2, u2, len(t_b[1]))
    assert np.mean(nc_a[0] + nc_b[0]) > 1.0


def test_batched_acceptance_statistics_match_oracle(orc):
    cfg = model_config("tiny", n_gen=128, batch=2)
    cfg["max_seq"] = 2048  # the faster image runs on while the slower one reaches 128 tokens
    wt, p0 = setup(cfg, wseed=101, pseed=102)
    p1 = prompt_tokens(dict(cfg, n_prompt=11), 103)
    eng = make_engine(cfg, weights_device(wt))
    gpu = [[], []]
    for s in range(10):
        eng.prefill_image(0, p0.cuda(), 500 + s)
        eng.prefill_image(1, p1.cuda(), 600 + s)
        ncs = [[], []]
        while min(sum(c) for c in ncs) < 128:
            _, nc1, _ = run_steps(eng, cfg, 2, 1, seed=700 + s, top_k=0)
            for b in range(2):
                ncs[b] += nc1[b]
        for b in range(2):
            # the image's steps until it had its 128 tokens
            k = int(np.searchsorted(np.cumsum(ncs[b]), 128)) + 1
            gpu[b] += ncs[b][:k]
    eng.close()
    m = orc.Model(cfg, weights_numpy(wt), max_seq=cfg["max_seq"])
    ocfg = orc.ModelCfg(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"],
                        cfg["ffn_dim"], cfg["vocab_size"], cfg["vis_lo"], cfg["V"], cfg["max_seq"], 1e-5, 1e4)
    for b, p in enumerate((p0, p1)):
        orc_nc = []
        for s in range(10):
            g = orc.gen_cfg(L=cfg["L"], V=cfg["V"], K=cfg["K"], D=cfg["D"], top_k=0, seed=800 + 10 * b + s,
                            n_prompt=len(p), n_gen=128, mcfg=ocfg, weights=m.w)
            _, steps, hist = orc.generate(g, p.numpy().astype(np.int32))
            orc_nc += sum(([i] * int(c) for i, c in enumerate(hist)), [])
        a, o = np.array(gpu[b], float), np.array(orc_nc, float)
        se = np.sqrt(a.var() / a.size + o.var() / o.size)
        print(f"image {b}: mean n_c gpu {a.mean():.3f} ({a.size} steps) oracle {o.mean():.3f} ({o.size}) se {se:.3f}")
        assert abs(a.mean() - o.mean()) < 4 * se + 0.02
    m.close()
