"""ctypes binding of the oracle library (plain C, see oracle.h).

TEST INFRASTRUCTURE: only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module. The product path never does.
"""
import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

TAG_ACC, TAG_RES, TAG_FRESH, TAG_BONUS, TAG_PD, TAG_INIT = 1, 2, 3, 4, 5, 6
AC, PD = 1, 2


class VerifyCfg(C.Structure):
    _fields_ = [("B", C.c_int32), ("L", C.c_int32), ("V", C.c_int32), ("K", C.c_int32),
                ("D", C.c_int32), ("top_k", C.c_int32), ("T", C.c_float), ("flags", C.c_uint32),
                ("seed", C.c_uint64), ("step", C.c_uint32), ("vis_lo", C.c_int32),
                ("eol_id", C.c_int32), ("row_len", C.c_int32), ("trial0", C.c_uint32)]


class VerifyIO(C.Structure):
    _fields_ = [("cur", C.c_void_p), ("draft", C.c_void_p), ("draft_tok", C.c_void_p),
                ("sib", C.c_void_p), ("in_meta", C.c_void_p), ("out_meta", C.c_void_p),
                ("out_tok", C.c_void_p), ("out_next", C.c_void_p), ("out_sib", C.c_void_p),
                ("out_rows", C.c_void_p), ("out_margin", C.c_void_p), ("dbg_p", C.c_void_p)]


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab_size", C.c_int32), ("vis_lo", C.c_int32), ("V", C.c_int32),
                ("max_seq", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float)]


class Weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("layer", C.c_void_p), ("final_norm", C.c_void_p),
                ("lm_head", C.c_void_p), ("is_f32", C.c_int32)]


class GenCfg(C.Structure):
    _fields_ = [("v", VerifyCfg), ("n_prompt", C.c_int32), ("n_gen", C.c_int32),
                ("max_steps", C.c_int32), ("mcfg", C.c_void_p), ("w", C.c_void_p),
                ("toy_V", C.c_int32), ("toy_salt", C.c_uint64),
                ("cfg_w", C.c_float), ("uncond", C.c_void_p), ("n_uncond", C.c_int32),
                ("step_meta", C.c_void_p), ("kv", C.c_void_p), ("kv_u", C.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from .build import build
            build()
        _lib = C.CDLL(LIB_PATH)
        _lib.orc_bits.restype = C.c_uint32
        _lib.orc_bits.argtypes = [C.c_uint64] + [C.c_uint32] * 6
        _lib.orc_uniform.restype = C.c_float
        _lib.orc_uniform.argtypes = [C.c_uint32]
        _lib.orc_exp1.restype = C.c_float
        _lib.orc_exp1.argtypes = [C.c_uint32]
        _lib.orc_topk_softmax.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_float, C.c_void_p]
        _lib.orc_race.argtypes = [C.c_void_p, C.c_int, C.c_uint64] + [C.c_uint32] * 5 + [C.c_void_p]
        _lib.orc_race_topn.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_uint64] + \
            [C.c_uint32] * 5 + [C.c_void_p, C.c_void_p]
        _lib.orc_race_many.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_uint64] + [C.c_uint32] * 4 + \
            [C.c_int, C.c_void_p]
        _lib.orc_race_many_ranked.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_uint64] + \
            [C.c_uint32] * 4 + [C.c_int, C.c_void_p]
        _lib.orc_race_ranked.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_uint64] + [C.c_uint32] * 5 + \
            [C.c_void_p]
        _lib.orc_race_topn_ranked.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_uint64] + \
            [C.c_uint32] * 5 + [C.c_void_p, C.c_void_p]
        _lib.orc_kv_row.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_void_p]
        _lib.orc_verify.argtypes = [C.POINTER(VerifyCfg), C.POINTER(VerifyIO)]
        _lib.orc_kv_new.restype = C.c_void_p
        _lib.orc_kv_new.argtypes = [C.POINTER(ModelCfg)]
        _lib.orc_cfg_combine.argtypes = [C.c_void_p, C.c_void_p, C.c_float, C.c_long, C.c_void_p]
        _lib.orc_kv_free.argtypes = [C.c_void_p]
        _lib.orc_kv_move.argtypes = [C.c_void_p, C.c_int, C.c_int]
        _lib.orc_forward.argtypes = [C.POINTER(ModelCfg), C.POINTER(Weights), C.c_void_p, C.c_int,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_int, C.c_void_p]
        _lib.orc_toy_logits.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_uint64, C.c_void_p]
        _lib.orc_generate.argtypes = [C.POINTER(GenCfg), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        _lib.orc_generate_many.argtypes = [C.POINTER(GenCfg), C.c_void_p, C.c_int, C.c_uint64,
                                           C.c_void_p, C.c_void_p, C.c_void_p]
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def philox(ctr, key):
    c = (C.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (C.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (C.c_uint32 * 4)()
    lib().orc_philox4x32_10(c, k, o)
    return [int(v) for v in o]


def bits(seed, tag, stage, row, trial, step, x):
    return int(lib().orc_bits(seed, tag, stage, row, trial, step, x))


def uniform(b):
    return float(lib().orc_uniform(b))


def topk_softmax(logits, top_k, T=1.0):
    l = np.ascontiguousarray(logits, dtype=np.float32)
    p = np.zeros_like(l)
    if lib().orc_topk_softmax(_p(l), l.size, int(top_k), C.c_float(T), _p(p)) != 0:
        raise ValueError("orc_topk_softmax: bad arguments")
    return p


def race(w, seed, tag, stage, row, trial, step):
    w = np.ascontiguousarray(w, dtype=np.float32)
    gap = np.zeros(1, np.float32)
    x = lib().orc_race(_p(w), w.size, seed, tag, stage, row, trial, step, _p(gap))
    return int(x), float(gap[0])


def race_topn(w, n, excl, seed, tag, stage, row, trial, step):
    w = np.ascontiguousarray(w, dtype=np.float32)
    out = np.zeros(max(n, 1), np.int32)
    gap = np.zeros(1, np.float32)
    lib().orc_race_topn(_p(w), w.size, n, excl, seed, tag, stage, row, trial, step, _p(out), _p(gap))
    return out[:n], float(gap[0])


def race_many(w, n, trials, seed=0, tag=TAG_RES, stage=0, row=0, step=0):
    """Independent races for trials 0..trials-1: [trials] winners (n <= 1) or
    [trials, n] ordered draws without replacement."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    out = np.zeros((trials, max(n, 1)), np.int32)
    lib().orc_race_many(_p(w), w.size, n, seed, tag, stage, row, step, trials, _p(out))
    return out[:, 0] if n <= 1 else out


def race_many_ranked(w, rank, n, trials, seed=0, tag=TAG_RES, stage=0, row=0, step=0):
    """race_many with the exponential of token x taken from stream element
    rank[x] (rank int32 [V], -1 for tokens that take no part)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    rank = np.ascontiguousarray(rank, dtype=np.int32)
    assert rank.size == w.size
    out = np.zeros((trials, max(n, 1)), np.int32)
    lib().orc_race_many_ranked(_p(w), _p(rank), w.size, n, seed, tag, stage, row, step, trials, _p(out))
    return out[:, 0] if n <= 1 else out


def race_ranked(w, rank, seed, tag, stage, row, trial, step):
    w = np.ascontiguousarray(w, dtype=np.float32)
    rank = np.ascontiguousarray(rank, dtype=np.int32)
    gap = np.zeros(1, np.float32)
    x = lib().orc_race_ranked(_p(w), _p(rank), w.size, seed, tag, stage, row, trial, step, _p(gap))
    return int(x), float(gap[0])


def race_topn_ranked(w, rank, n, excl, seed, tag, stage, row, trial, step):
    w = np.ascontiguousarray(w, dtype=np.float32)
    rank = np.ascontiguousarray(rank, dtype=np.int32)
    out = np.zeros(max(n, 1), np.int32)
    gap = np.zeros(1, np.float32)
    lib().orc_race_topn_ranked(_p(w), _p(rank), w.size, n, excl, seed, tag, stage, row, trial, step, _p(out),
                               _p(gap))
    return out[:n], float(gap[0])


def verify(cur, draft, draft_tok, in_meta, *, K, D, top_k, T=1.0, flags=AC | PD, seed=0, step=0,
           sib=None, vis_lo=0, eol_id=-1, row_len=0, want_p=False, trial0=0):
    """One verification step over B trials. Arrays: cur/draft [B,L,V] f32,
    draft_tok [B,L] i32, in_meta [B,4] i32, sib [B,D,K-1] i32 or None."""
    cur = np.ascontiguousarray(cur, dtype=np.float32)
    B, L, V = cur.shape
    draft = np.ascontiguousarray(draft, dtype=np.float32)
    draft_tok = np.ascontiguousarray(draft_tok, dtype=np.int32)
    in_meta = np.ascontiguousarray(in_meta, dtype=np.int32)
    if sib is not None:
        sib = np.ascontiguousarray(sib, dtype=np.int32)
        assert sib.shape == (B, D, K - 1)
    out = {
        "meta": np.zeros((B, 8), np.int32),
        "tok": np.zeros((B, L), np.int32),
        "next": np.zeros((B, L), np.int32),
        "sib": np.zeros((B, max(D, 1), max(K - 1, 1)), np.int32)[:, :D, :K - 1].copy(),
        "rows": np.zeros((B, L, 2), np.int32),
        "margin": np.zeros((B, L, 4), np.float32),
    }
    dbg = np.zeros((B, L, V), np.float32) if want_p else None
    cfg = VerifyCfg(B, L, V, K, D, top_k, T, flags, seed, step, vis_lo, eol_id, row_len, trial0)
    io = VerifyIO(_p(cur), _p(draft), _p(draft_tok), _p(sib), _p(in_meta), _p(out["meta"]),
                  _p(out["tok"]), _p(out["next"]), _p(out["sib"]), _p(out["rows"]),
                  _p(out["margin"]), _p(dbg))
    rc = lib().orc_verify(C.byref(cfg), C.byref(io))
    if rc != 0:
        raise ValueError(f"orc_verify failed: {rc}")
    if want_p:
        out["p"] = dbg
    return out


def toy_logits(ctx, V, salt):
    ctx = np.ascontiguousarray(ctx, dtype=np.int32)
    out = np.zeros(V, np.float32)
    lib().orc_toy_logits(_p(ctx), ctx.size, V, salt, _p(out))
    return out


def cfg_combine(l_c, l_u, w):
    """Classifier-free guidance l_u + w (l_c - l_u) (Sec. 5.1), fp64 rounded once."""
    l_c = np.ascontiguousarray(l_c, dtype=np.float32)
    l_u = np.ascontiguousarray(l_u, dtype=np.float32)
    assert l_c.shape == l_u.shape
    out = np.empty_like(l_c)
    lib().orc_cfg_combine(_p(l_c), _p(l_u), w, l_c.size, _p(out))
    return out


def gen_cfg(*, L, V, K, D, top_k=0, T=1.0, flags=AC | PD, seed=0, n_prompt, n_gen, max_steps=100000,
            toy_salt=0, vis_lo=0, eol_id=-1, row_len=0, mcfg=None, weights=None, cfg_w=0.0, uncond=None):
    """Generation config. With cfg_w != 0 (transformer only), `uncond` is the
    unconditional prompt (kept alive on the returned object)."""
    vc = VerifyCfg(1, L, V, K, D, top_k, T, flags, seed, 0, vis_lo, eol_id, row_len, 0)
    u = None if uncond is None else np.ascontiguousarray(uncond, dtype=np.int32)
    g = GenCfg(vc, n_prompt, n_gen, max_steps,
               C.addressof(mcfg) if mcfg is not None else None,
               C.addressof(weights) if weights is not None else None,
               V if mcfg is None else 0, toy_salt, cfg_w, _p(u) if u is not None else None,
               0 if u is None else u.size)
    g._uncond = u
    return g


def generate_many(cfg, prompt, runs, seed0):
    prompt = np.ascontiguousarray(prompt, dtype=np.int32)
    out = np.zeros((runs, cfg.n_gen), np.int32)
    steps = np.zeros(runs, np.int32)
    hist = np.zeros(cfg.v.L + 2, np.int64)
    rc = lib().orc_generate_many(C.byref(cfg), _p(prompt), runs, seed0, _p(out), _p(steps), _p(hist))
    if rc != 0:
        raise RuntimeError("orc_generate_many failed")
    return out, steps, hist


def generate(cfg, prompt, step_meta=False, model=None, model_u=None):
    """One generation. With step_meta, also returns every step's out-meta
    [steps, 8]; with model (and model_u for the unconditional stream of a
    guided generation), the generation runs on that Model's cache, which then
    holds the final cache."""
    prompt = np.ascontiguousarray(prompt, dtype=np.int32)
    out = np.zeros(cfg.n_gen + 2 * cfg.v.L + 2, np.int32)
    steps = np.zeros(1, np.int32)
    hist = np.zeros(cfg.v.L + 2, np.int64)
    sm = np.zeros((cfg.max_steps, 8), np.int32) if step_meta else None
    cfg.step_meta = _p(sm)
    cfg.kv = model.kv if model is not None else None
    cfg.kv_u = model_u.kv if model_u is not None else None
    try:
        g = lib().orc_generate(C.byref(cfg), _p(prompt), _p(out), _p(steps), _p(hist))
    finally:
        cfg.step_meta = None
        cfg.kv = None
        cfg.kv_u = None
    if g < 0:
        raise RuntimeError("orc_generate failed")
    if step_meta:
        return out[:g], int(steps[0]), hist, sm[:int(steps[0])]
    return out[:g], int(steps[0]), hist


class Model:
    """Holds model config + weights (numpy arrays, bf16 as uint16 or f32) and
    an oracle KV cache."""

    def __init__(self, cfg: dict, weights: dict, max_seq: int):
        self.cfg = ModelCfg(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"],
                            cfg["head_dim"], cfg["ffn_dim"], cfg["vocab_size"], cfg["vis_lo"],
                            cfg["V"], max_seq, cfg.get("rms_eps", 1e-5), cfg.get("rope_theta", 1e4))
        self._keep = []
        is_f32 = weights["embed"].dtype == np.float32

        def ptr(a):
            a = np.ascontiguousarray(a)
            assert (a.dtype == np.float32) == is_f32
            self._keep.append(a)
            return a.ctypes.data

        names = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"]
        layer_ptrs = (C.c_void_p * (9 * cfg["n_layers"]))()
        for l in range(cfg["n_layers"]):
            for i, nm in enumerate(names):
                layer_ptrs[9 * l + i] = ptr(weights["layers"][l][nm])
        self._layer_ptrs = layer_ptrs
        self.w = Weights(ptr(weights["embed"]), C.cast(layer_ptrs, C.c_void_p).value,
                         ptr(weights["final_norm"]), ptr(weights["lm_head"]), 1 if is_f32 else 0)
        self.kv = lib().orc_kv_new(C.byref(self.cfg))
        if not self.kv:
            raise MemoryError("orc_kv_new")

    def forward(self, n, tok, pos, anc, logits=True):
        tok = np.ascontiguousarray(tok, dtype=np.int32)
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        anc = np.ascontiguousarray(anc, dtype=np.uint64)
        M = tok.size
        out = np.zeros((M, self.cfg.V), np.float32) if logits else None
        rc = lib().orc_forward(C.byref(self.cfg), C.byref(self.w), self.kv, n, _p(tok), _p(pos), _p(anc),
                               M, _p(out))
        if rc != 0:
            raise ValueError(f"orc_forward failed: {rc}")
        return out

    def kv_move(self, src, dst):
        lib().orc_kv_move(self.kv, src, dst)

    def kv_row(self, layer, row):
        """(key, value) of cache row `row` in layer `layer`, float64 [Hkv*hd] each."""
        n = self.cfg.n_kv_heads * self.cfg.head_dim
        k = np.zeros(n, np.float64)
        v = np.zeros(n, np.float64)
        lib().orc_kv_row(self.kv, layer, row, _p(k), _p(v))
        return k, v

    def close(self):
        if self.kv:
            lib().orc_kv_free(self.kv)
            self.kv = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
