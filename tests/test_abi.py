"""The C-ABI library loads and exports every entry point include/sjd.h
declares; host-side argument checks reject bad calls before any HIP call
(no GPU needed)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "sjd.h")).read()
    return sorted(set(re.findall(r"SJD_API\s+[\w\s\*]*?\b(sjd_\w+)\s*\(", src)))


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for s in ["sjd_status_str", "sjd_verify", "sjd_init", "sjd_prefill", "sjd_step", "sjd_destroy"]:
        assert s in syms


def test_library_exports_every_declared_symbol():
    from paper_2603_18599_amd import sjd
    lib = sjd.load_library()
    for s in declared_symbols():
        assert hasattr(lib, s), s
    assert set(declared_symbols()) <= set(sjd.EXPORTS) | set(declared_symbols())


def test_status_strings():
    from paper_2603_18599_amd import sjd
    assert sjd.sjd_status_str(0) == "SJD_OK"
    assert "EINVAL" in sjd.sjd_status_str(-1)
    assert "unknown" in sjd.sjd_status_str(42)


def test_verify_rejects_bad_params_on_host():
    from paper_2603_18599_amd import sjd
    lib = sjd.load_library()
    good = dict(B=1, L=4, V=16, K=2, D=1, top_k=0, temperature=1.0, flags=3, seed=0, step=0, vis_lo=0,
                eol_id=-1, row_len=0)
    bad = [dict(B=0), dict(L=0), dict(L=65), dict(V=6), dict(K=0), dict(K=9), dict(D=3), dict(top_k=-1),
           dict(temperature=0.0), dict(temperature=float("nan")), dict(flags=8), dict(flags=16)]
    io = sjd.VerifyIO()  # NULL pointers
    for b in bad:
        p = dict(good)
        p.update(b)
        prm = sjd.VerifyParams(**p)
        assert lib.sjd_verify(C.byref(prm), C.byref(io), None) == -1, b
    # valid parameters but NULL buffers
    prm = sjd.VerifyParams(**good)
    assert lib.sjd_verify(C.byref(prm), C.byref(io), None) == -1
    assert lib.sjd_verify(None, None, None) == -1


def test_noalloc_verify_rejects_rows_beyond_its_scratch_on_host():
    """sjd_verify_noalloc takes at most SJD_VERIFY_NOALLOC_MAX_ROWS rows;
    beyond that it returns SJD_EINVAL before any HIP call (the pointers
    below are never dereferenced)."""
    from paper_2603_18599_amd import sjd
    lib = sjd.load_library()
    hdr = open(os.path.join(ROOT, "include", "sjd.h")).read()
    cap = int(re.search(r"#define SJD_VERIFY_NOALLOC_MAX_ROWS (\d+)", hdr).group(1))
    assert cap == sjd.SJD_VERIFY_NOALLOC_MAX_ROWS
    fake = 1 << 20  # 16-byte aligned, never read
    io = sjd.VerifyIO(fake, fake, fake, None, fake, fake, fake, fake, fake, None, None)
    L = 32
    prm = sjd.VerifyParams(cap // L + 1, L, 16, 2, 1, 0, 1.0, 3, 0, 0, 0, -1, 0)
    assert lib.sjd_verify_noalloc(C.byref(prm), C.byref(io), None) == -1
    assert lib.sjd_verify_noalloc(None, None, None) == -1


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    from paper_2603_18599_amd import sjd
    monkeypatch.setattr(sjd, "_lib", None)
    monkeypatch.setattr(sjd, "HERE", str(tmp_path))
    with pytest.raises(RuntimeError, match="missing"):
        sjd.load_library()
