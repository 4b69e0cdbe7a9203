"""ctypes binding of libsjd.so (include/sjd.h): argument marshalling only.

Device buffers are torch tensors on the current HIP device; their data
pointers and the current torch stream are handed to the C entry points.
Every step of the computation runs in the library's HIP kernels; there is no
fallback path.
"""
import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libsjd.so"

SJD_AC = 1
SJD_PD = 2
SJD_EAGER = 4
SJD_NO_TUNE = 8
SJD_TUNE = 16
SJD_CHECK_FINITE = 32
SJD_FULL_SELECT = 64
SJD_VERIFY_NOALLOC_MAX_ROWS = 131072

_STATUS = {0: "SJD_OK", -1: "SJD_EINVAL", -2: "SJD_ENOMEM", -3: "SJD_EHIP", -4: "SJD_ESTATE", -5: "SJD_ENOTSUP",
           -6: "SJD_ENONFINITE"}


class SjdError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} failed: {_STATUS.get(code, code)}")
        self.code = code


class VerifyParams(C.Structure):
    _fields_ = [("B", C.c_int32), ("L", C.c_int32), ("V", C.c_int32), ("K", C.c_int32), ("D", C.c_int32),
                ("top_k", C.c_int32), ("temperature", C.c_float), ("flags", C.c_uint32), ("seed", C.c_uint64),
                ("step", C.c_uint32), ("vis_lo", C.c_int32), ("eol_id", C.c_int32), ("row_len", C.c_int32)]


class VerifyIO(C.Structure):
    _fields_ = [("d_cur", C.c_void_p), ("d_draft", C.c_void_p), ("d_draft_tok", C.c_void_p),
                ("d_sib", C.c_void_p), ("d_in_meta", C.c_void_p), ("d_out_meta", C.c_void_p),
                ("d_out_tok", C.c_void_p), ("d_out_next", C.c_void_p), ("d_out_sib", C.c_void_p),
                ("d_out_rows", C.c_void_p), ("d_dbg_p", C.c_void_p)]


class Config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab_size", C.c_int32), ("vis_lo", C.c_int32), ("V", C.c_int32), ("max_seq", C.c_int32),
                ("L", C.c_int32), ("K", C.c_int32), ("D", C.c_int32), ("flags", C.c_uint32),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float), ("eol_id", C.c_int32),
                ("row_len", C.c_int32), ("weights_f32", C.c_int32), ("cfg_w", C.c_float),
                ("batch", C.c_int32)]


class Weights(C.Structure):
    _fields_ = [("d_embed", C.c_void_p), ("h_layer", C.c_void_p), ("d_final_norm", C.c_void_p),
                ("d_lm_head", C.c_void_p)]


EXPORTS = ["sjd_status_str", "sjd_verify", "sjd_verify_noalloc", "sjd_init", "sjd_prefill", "sjd_prefill_image",
           "sjd_prefill_cfg", "sjd_prefill_image_cfg", "sjd_set_drafts", "sjd_step", "sjd_forward_window",
           "sjd_get_plan", "sjd_destroy"]

_lib = None


def lib_path():
    """The in-tree library, or the one SJD_LIBRARY names (another build of
    the same sources, e.g. to compare two builds in one process tree)."""
    return os.environ.get("SJD_LIBRARY") or os.path.join(HERE, _LIB_NAME)


def load_library():
    """Loads libsjd.so (built in-tree by __graft_entry__.build()); raises if
    it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build the HIP library first (python -c "
                           "'import __graft_entry__ as g; g.build()')")
    lib = C.CDLL(path)
    lib.sjd_status_str.restype = C.c_char_p
    lib.sjd_status_str.argtypes = [C.c_int]
    lib.sjd_verify.restype = C.c_int
    lib.sjd_verify.argtypes = [C.POINTER(VerifyParams), C.POINTER(VerifyIO), C.c_void_p]
    lib.sjd_verify_noalloc.restype = C.c_int
    lib.sjd_verify_noalloc.argtypes = [C.POINTER(VerifyParams), C.POINTER(VerifyIO), C.c_void_p]
    lib.sjd_init.restype = C.c_int
    lib.sjd_init.argtypes = [C.POINTER(Config), C.POINTER(Weights), C.c_void_p, C.POINTER(C.c_void_p)]
    lib.sjd_prefill.restype = C.c_int
    lib.sjd_prefill.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_uint64, C.c_void_p]
    lib.sjd_get_plan.restype = C.c_int
    lib.sjd_get_plan.argtypes = [C.c_void_p, C.POINTER(C.c_int32), C.c_int32]
    lib.sjd_prefill_image.restype = C.c_int
    lib.sjd_prefill_image.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_uint64, C.c_void_p]
    lib.sjd_prefill_cfg.restype = C.c_int
    lib.sjd_prefill_cfg.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_uint64,
                                    C.c_void_p]
    lib.sjd_prefill_image_cfg.restype = C.c_int
    lib.sjd_prefill_image_cfg.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_int32, C.c_void_p, C.c_int32,
                                          C.c_uint64, C.c_void_p]
    lib.sjd_step.restype = C.c_int
    lib.sjd_step.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_float, C.c_int32,
                             C.c_uint64, C.c_uint32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.sjd_set_drafts.restype = C.c_int
    lib.sjd_set_drafts.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.sjd_forward_window.restype = C.c_int
    lib.sjd_forward_window.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
    lib.sjd_destroy.restype = None
    lib.sjd_destroy.argtypes = [C.c_void_p]
    _lib = lib
    return lib


def sjd_status_str(code):
    return load_library().sjd_status_str(code).decode()


def _ptr(t):
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _check(fn, rc):
    if rc != 0:
        raise SjdError(fn, rc)


def sjd_verify(cur, draft, draft_tok, in_meta, out, *, K, D, top_k, temperature=1.0, flags=SJD_AC | SJD_PD,
               seed=0, step=0, sib=None, vis_lo=0, eol_id=-1, row_len=0, out_rows=None, dbg_p=None, stream=None,
               noalloc=False):
    """Standalone verification (sjd_verify in include/sjd.h; noalloc:
    sjd_verify_noalloc). cur/draft: float32 [B,L,V] device tensors; draft_tok
    int32 [B,L]; in_meta int32 [B,4]; out: dict of int32 device tensors meta
    [B,8], tok [B,L], next [B,L], sib [B,D,K-1]."""
    B, L, V = cur.shape
    p = VerifyParams(B, L, V, K, D, top_k, temperature, flags, seed, step, vis_lo, eol_id, row_len)
    io = VerifyIO(_ptr(cur), _ptr(draft), _ptr(draft_tok), _ptr(sib), _ptr(in_meta), _ptr(out["meta"]),
                  _ptr(out["tok"]), _ptr(out["next"]), _ptr(out["sib"]), _ptr(out_rows), _ptr(dbg_p))
    lib = load_library()
    fn = "sjd_verify_noalloc" if noalloc else "sjd_verify"
    _check(fn, getattr(lib, fn)(C.byref(p), C.byref(io), _stream(stream)))


def verify_outputs(B, L, K, D, device="cuda"):
    import torch
    return {"meta": torch.zeros(B, 8, dtype=torch.int32, device=device),
            "tok": torch.zeros(B, L, dtype=torch.int32, device=device),
            "next": torch.zeros(B, L, dtype=torch.int32, device=device),
            "sib": torch.zeros(B, max(D, 0), max(K - 1, 0), dtype=torch.int32, device=device)}


class Engine:
    """A decoder context (sjd_init .. sjd_destroy)."""

    def __init__(self, cfg: dict, weights: dict, stream=None):
        lib = load_library()
        self.cfg = cfg
        c = Config(cfg["n_layers"], cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"],
                   cfg["ffn_dim"], cfg["vocab_size"], cfg["vis_lo"], cfg["V"], cfg["max_seq"], cfg["L"], cfg["K"],
                   cfg["D"], cfg.get("flags", SJD_AC | SJD_PD), cfg.get("rms_eps", 1e-5),
                   cfg.get("rope_theta", 1e4), cfg.get("eol_id", -1), cfg.get("row_len", 0),
                   1 if cfg.get("weights_f32", False) else 0, cfg.get("cfg_w", 0.0), cfg.get("batch", 1))
        names = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"]
        self._layer_ptrs = (C.c_void_p * (9 * cfg["n_layers"]))()
        for l in range(cfg["n_layers"]):
            for i, nm in enumerate(names):
                self._layer_ptrs[9 * l + i] = weights["layers"][l][nm].data_ptr()
        self._weights = weights  # keep alive
        w = Weights(weights["embed"].data_ptr(), C.cast(self._layer_ptrs, C.c_void_p).value,
                    weights["final_norm"].data_ptr(), weights["lm_head"].data_ptr())
        h = C.c_void_p()
        _check("sjd_init", lib.sjd_init(C.byref(c), C.byref(w), _stream(stream), C.byref(h)))
        self.h = h

    def prefill(self, prompt, seed, stream=None):
        _check("sjd_prefill", load_library().sjd_prefill(self.h, _ptr(prompt), prompt.numel(), seed,
                                                          _stream(stream)))

    def plan(self, rows64=False):
        """GEMM plan chosen at init for windows of up to 32 rows (or, rows64,
        of more): splits [qkv, o, gate|up, down, head] followed by the column
        blocks per workgroup of each."""
        out = (C.c_int32 * 20)()
        _check("sjd_get_plan", load_library().sjd_get_plan(self.h, out, 20))
        return list(out)[10:] if rows64 else list(out)[:10]

    def plan_pin(self):
        """The plan for windows of up to 32 rows as an SJD_SPLITS value."""
        p = self.plan()
        return ",".join(f"{p[i]}:{p[5 + i]}" for i in range(4))

    def prefill_image(self, image, prompt, seed, stream=None):
        """Batched contexts: (re)starts image `image` with `prompt`."""
        _check("sjd_prefill_image", load_library().sjd_prefill_image(self.h, image, _ptr(prompt), prompt.numel(), seed,
                                                                      _stream(stream)))

    def prefill_cfg(self, prompt, uncond, seed, stream=None, image=None):
        """Guided contexts (cfg_w != 0): text prompt and unconditional prompt
        (of image `image` of a guided batch; None: sjd_prefill_cfg)."""
        lib = load_library()
        if image is None:
            _check("sjd_prefill_cfg", lib.sjd_prefill_cfg(self.h, _ptr(prompt), prompt.numel(), _ptr(uncond),
                                                          uncond.numel(), seed, _stream(stream)))
        else:
            _check("sjd_prefill_image_cfg", lib.sjd_prefill_image_cfg(self.h, image, _ptr(prompt), prompt.numel(),
                                                                      _ptr(uncond), uncond.numel(), seed,
                                                                      _stream(stream)))

    def set_drafts(self, draft_tok, draft_logits=None, image=0, stream=None):
        """The next step verifies draft_tok (int32 [L], vocabulary ids) against
        draft_logits (float32 [L][V] logits over the sampled range, or None)."""
        _check("sjd_set_drafts", load_library().sjd_set_drafts(self.h, image, _ptr(draft_tok), _ptr(draft_logits),
                                                                _stream(stream)))

    def step(self, temperature, top_k, seed, step, out_meta=None, out_tok=None, out_next=None, stream=None,
             draft_tok=None, draft_logits=None):
        """One iteration. draft_tok (int32 [batch, L] vocabulary ids) and
        draft_logits (float32 [batch, L, V] or None) replace the context's
        own drafts for this step (None: the context's)."""
        _check("sjd_step", load_library().sjd_step(self.h, _ptr(draft_tok), _ptr(draft_logits), 0, 0, temperature,
                                                    top_k, seed, step, _ptr(out_meta), _ptr(out_tok),
                                                    _ptr(out_next), _stream(stream)))

    def forward_window(self, logits, stream=None):
        _check("sjd_forward_window", load_library().sjd_forward_window(self.h, _ptr(logits), _stream(stream)))

    def close(self):
        if getattr(self, "h", None):
            load_library().sjd_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
