"""The pins have teeth: plausible mistakes planted in a copy of the oracle's
sources (a dropped term, a transposed operand, a wrong row or offset, a
missing break) must each make one of the pin tests fail.

Each case copies oracle/*.c to a temporary directory, applies one textual
edit, builds that copy, points the oracle binding at it, runs a pin test and
expects it to fail. The committed oracle is never modified.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import test_oracle_forward as tf
import test_oracle_kv as tk
import test_oracle_sequence as ts
import test_oracle_verify as tv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORC = os.path.join(ROOT, "oracle")


def build_planted(tmp, fname, old, new):
    for f in os.listdir(ORC):
        if f.endswith((".c", ".h")):
            shutil.copy(os.path.join(ORC, f), tmp)
    path = os.path.join(tmp, fname)
    src = open(path).read()
    assert src.count(old) == 1, f"plant anchor not found exactly once in {fname}: {old!r}"
    open(path, "w").write(src.replace(old, new))
    lib = os.path.join(tmp, "liboracle.so")
    srcs = [os.path.join(tmp, s) for s in ("rng.c", "verify.c", "forward.c", "generate.c")]
    subprocess.run(["gcc", "-std=c11", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared", "-o", lib]
                   + srcs + ["-lm"], check=True, capture_output=True)
    return lib


def seq_law(orc, **kw):
    pval, _, _ = ts.check_law(orc, runs=200_000, **kw)
    assert pval > 1e-4, pval


def single(orc):
    tv.test_single_draft_lossless_and_acceptance(orc, "random")


def kcand(orc):
    tv.test_k_candidates_without_replacement_lossless(orc, 3)


def forward_torch(orc):
    wt = tf.make_weights(tf.CFG, 1)
    m = orc.Model(tf.CFG, tf.to_numpy(wt), max_seq=64)
    try:
        tf.test_forward_matches_torch_reference((m, wt))
        tf.test_forward_tree_mask_matches_torch((m, wt))
    finally:
        m.close()


PLANTS = {
    # residual drawn from p instead of max(0, p - q)
    "residual_drops_q": ("verify.c", "float r = py - qy;", "float r = py;", single),
    # accept ratio transposed
    "ratio_transposed": ("verify.c", "float ratio = pk / qk;", "float ratio = qk / pk;", single),
    # q^(k) neither excludes rejected candidates nor renormalises
    "qk_not_renormalised": ("verify.c", "float qy = (excl[y] || !(den > 0.0f)) ? 0.0f : q[y] / den;",
                            "float qy = q[y];", kcand),
    # candidate k > 1 checked against the stage-1 ratio
    "pk_not_renormalised": ("verify.c", "float pk = rho[x] / Nf;", "float pk = p[x];", kcand),
    # first-rejection break dropped: r becomes the last rejected row
    "no_break_in_first_rej": ("verify.c", "if (!accepted) { r = j; break; }", "if (!accepted) { r = j; }",
                              lambda o: seq_law(o, L=4, K=2, D=1, flags=1)),
    # bonus after an accepted sibling taken from the spine row (stale context)
    "bonus_from_spine_row": ("verify.c", "int t = n_s + r * Km1 + (acc_k - 2);\n      otok[r] = ro[r].tok",
                             "int t = r + 1;\n      otok[r] = ro[r].tok",
                             lambda o: seq_law(o, L=4, K=2, D=2, flags=3)),
    # next step's q rows shifted by one
    "q_rows_off_by_one": ("generate.c", "q_off = n_c;", "q_off = n_c - 1;",
                          lambda o: seq_law(o, L=4, K=2, D=1, flags=1)),
    # drafts carried over from the wrong row
    "carry_wrong_row": ("verify.c", "    int j = n_c + i;\n    long g = g0 + n_c + i;",
                        "    int j = n_c + i + 1 < n_s ? n_c + i + 1 : n_c + i;\n    long g = g0 + n_c + i;",
                        lambda o: seq_law(o, L=4, K=2, D=1, flags=1)),
    # window mask taken as plain causal order, ignoring the tree
    "mask_ignores_tree": ("forward.c", "int vis = t < n || ((anc[a] >> (t - n)) & 1u);",
                          "int vis = t < n || (t - n <= a);", forward_torch),
    # rotary sign slip
    "rope_sign": ("forward.c", "v[i] = a * cs - b * sn;", "v[i] = a * cs + b * sn;", forward_torch),
    # accepted sibling's key/value row moved one row short (onto the last kept spine row)
    "kv_move_dest_off_by_one": ("generate.c", "orc_kv_move(kv, n + n_s + r * Km1 + (acc_k - 2), n + r + 1);",
                                "orc_kv_move(kv, n + n_s + r * Km1 + (acc_k - 2), n + r);",
                                lambda o: tk.test_cache_equals_recompute_after_sibling_commits(o, 0, 1.0, 8, 3, 2)),
    # the row of the neighbouring sibling moved instead of the accepted one
    "kv_move_wrong_sibling": ("generate.c", "orc_kv_move(kv, n + n_s + r * Km1 + (acc_k - 2), n + r + 1);",
                              "orc_kv_move(kv, n + n_s + r * Km1 + (acc_k - 2) + (acc_k == 2), n + r + 1);",
                              lambda o: tk.test_cache_equals_recompute_after_sibling_commits(o, 0, 1.0, 8, 3, 2)),
    # the unconditional stream's cache not backtracked
    "kv_move_guided_missing": ("generate.c", "if (cfg_on && acc_k >= 2) orc_kv_move(",
                               "if (0 && cfg_on && acc_k >= 2) orc_kv_move(",
                               lambda o: tk.test_guided_caches_equal_recompute_after_sibling_commits(o)),
    # a ranked race reads stream element x instead of the token's rank
    "race_ignores_rank": ("rng.c", "const uint32_t e_idx = rank ? (uint32_t)rank[x] : (uint32_t)x;\n    float e = orc_exp1",
                          "const uint32_t e_idx = (uint32_t)x;\n    float e = orc_exp1",
                          lambda o: __import__("test_oracle_rng").test_ranked_race_is_the_race_over_the_compact_list(o)),
    # tie order of the top-k set reversed
    "topk_tie_order": ("verify.c", "return (x->idx > y->idx) - (x->idx < y->idx);",
                       "return (x->idx < y->idx) - (x->idx > y->idx);", lambda o: tv.test_topk_tie_order(o)),
}


@pytest.mark.parametrize("name", sorted(PLANTS))
def test_planted_mistake_is_caught(orc, tmp_path, name):
    fname, old, new, check = PLANTS[name]
    lib = build_planted(str(tmp_path), fname, old, new)
    saved_lib, saved_path = orc._lib, orc.LIB_PATH
    try:
        orc._lib = None
        orc.LIB_PATH = lib
        orc.lib()
        with pytest.raises((AssertionError, ValueError, RuntimeError)):
            check(orc)
    finally:
        orc._lib, orc.LIB_PATH = saved_lib, saved_path
