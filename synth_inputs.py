"""Seeded synthetic inputs shared by the tests, the smoke check and the
benchmark (both the HIP path and the oracle consume them).

This module holds no arithmetic of the method: it only draws random logits,
draft tokens, prompts and weights with torch's seeded generators, shaped like
the paper's workloads (Lumina-mGPT 7B at 768x768 = 48x48 image tokens plus row
ends; Emu3 8B at 720x720 = 90x90 plus row ends; top-2000 sampling at
temperature 1; Sec. 5.1). Datasets and trained weights are not available, so
random prompt ids and random-init weights N(0, 0.02) stand in for them.
"""
import torch

# Workloads (decoder shapes, window, sampler).
CONFIGS = {
    "tiny": dict(n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=1024,
                 vocab_size=1024, vis_lo=0, V=1024, L=16, K=4, D=3, top_k=0, temperature=1.0,
                 n_prompt=16, n_gen=256, row_len=0, eol_id=-1, weights_f32=True),
    "verify": dict(B=4096, L=32, V=16384, K=4, D=3, top_k=2000, temperature=1.0, logit_std=2.0,
                   draft_noise=0.5),
    "mid": dict(n_layers=12, d_model=1024, n_heads=16, n_kv_heads=16, head_dim=64, ffn_dim=2816,
                vocab_size=16384, vis_lo=0, V=16384, L=32, K=4, D=3, top_k=2000, temperature=1.0,
                n_prompt=64, n_gen=1024, row_len=0, eol_id=-1, weights_f32=False),
    "7b": dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128, ffn_dim=11008,
               vocab_size=65536, vis_lo=0, V=65536, L=32, K=4, D=3, top_k=2000, temperature=1.0,
               n_prompt=64, n_gen=2352, row_len=48, eol_id=65535, weights_f32=False),
    "8b": dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128, ffn_dim=14336,
               vocab_size=184622, vis_lo=151854, V=32768, L=32, K=4, D=3, top_k=2048, temperature=1.0,
               n_prompt=64, n_gen=8190, row_len=90, eol_id=151853, weights_f32=False),
}


def model_config(name, **over):
    c = dict(CONFIGS[name])
    c.update(over)
    c.setdefault("max_seq", c["n_prompt"] + c["n_gen"] + 2 * c["L"] + 8)
    c.setdefault("rms_eps", 1e-5)
    c.setdefault("rope_theta", 1e4)
    return c


def verify_inputs(B, L, V, *, top_k, seed, logit_std=2.0, draft_noise=0.5, temperature=1.0, K=4, D=3, D_in=0,
                  n_q=None, device="cpu", int_logits=False):
    """Current logits ~ N(0, logit_std^2); draft logits = current + N(0,
    draft_noise^2); spine drafts (and, for D_in > 0, K-1 siblings at rows
    < D_in) drawn without replacement from top-k softmax of the draft logits
    by torch.multinomial. Returns a dict of tensors on `device`."""
    g = torch.Generator(device=device).manual_seed(seed)
    if int_logits:
        cur = torch.randint(-3, 4, (B, L, V), generator=g, device=device).float()
        draft = cur + torch.randint(-1, 2, (B, L, V), generator=g, device=device).float()
    else:
        cur = torch.randn(B, L, V, generator=g, device=device) * logit_std
        draft = cur + torch.randn(B, L, V, generator=g, device=device) * draft_noise
    k = V if top_k <= 0 or top_k >= V else top_k
    vals, idx = torch.topk(draft.view(B * L, V), k, dim=1)
    probs = torch.softmax(vals.double() / temperature, dim=1)
    nsamp = K if D_in > 0 else 1
    nsamp = min(nsamp, k)
    pick = torch.multinomial(probs, nsamp, replacement=False, generator=g)
    toks = torch.gather(idx, 1, pick).view(B, L, nsamp).to(torch.int32)
    draft_tok = toks[:, :, 0].contiguous()
    sib = None
    if D > 0 and K > 1:
        sib = torch.full((B, D, K - 1), -1, dtype=torch.int32, device=device)
        if D_in > 0:
            n = min(K - 1, nsamp - 1)
            sib[:, :D_in, :n] = toks[:, :D_in, 1:1 + n]
    n_s = L - (K - 1) * D_in
    if n_q is None:
        n_q = n_s
    meta = torch.zeros(B, 4, dtype=torch.int32, device=device)
    meta[:, 0] = D_in
    meta[:, 1] = n_q
    return dict(cur=cur.contiguous(), draft=draft.contiguous(), draft_tok=draft_tok, sib=sib, meta=meta)


def model_weights(cfg, seed, device="cpu", std=0.02):
    """Random-init decoder weights, row-major [out][in]: N(0, std^2) matrices,
    unit norm gains; bf16 unless cfg['weights_f32']."""
    g = torch.Generator(device=device).manual_seed(seed)
    dt = torch.float32 if cfg.get("weights_f32", False) else torch.bfloat16
    d, H, Hkv, hd, F, Vv = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim",
                                              "vocab_size"))

    def mat(o, i):
        t = torch.empty(o, i, device=device, dtype=torch.float32)
        t.normal_(0.0, std, generator=g)
        return t.to(dt)

    def ones(n):
        return torch.ones(n, device=device, dtype=dt)

    layers = []
    for _ in range(cfg["n_layers"]):
        layers.append(dict(attn_norm=ones(d), wq=mat(H * hd, d), wk=mat(Hkv * hd, d), wv=mat(Hkv * hd, d),
                           wo=mat(d, H * hd), ffn_norm=ones(d), wg=mat(F, d), wu=mat(F, d), wd=mat(d, F)))
    return dict(embed=mat(Vv, d), layers=layers, final_norm=ones(d), lm_head=mat(Vv, d))


def prompt_tokens(cfg, seed, device="cpu"):
    """Random prompt ids over the whole vocabulary (text prompts of a random
    model carry no meaning)."""
    g = torch.Generator(device=device).manual_seed(seed)
    return torch.randint(0, cfg["vocab_size"], (cfg["n_prompt"],), generator=g, device=device, dtype=torch.int32)


def image_history(cfg, n, seed, device="cpu"):
    """n already-generated image tokens: random visual ids in [vis_lo, vis_lo
    + V), the row-end id at every (row_len + 1)-th position (Lumina-mGPT and
    Emu3 end each image row with a row-end token). Stands in for the first part
    of an image so that a step can be timed at a mid-image cache length."""
    g = torch.Generator(device=device).manual_seed(seed)
    t = torch.randint(cfg["vis_lo"], cfg["vis_lo"] + cfg["V"], (n,), generator=g, device=device, dtype=torch.int32)
    if cfg.get("row_len", 0) > 0:
        t[cfg["row_len"]::cfg["row_len"] + 1] = cfg["eol_id"]
    return t

