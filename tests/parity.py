"""Comparison of sjd_verify (HIP) outputs with the oracle's, with the near-tie
classes of the parity bar:
  (i)   accept near-tie   |u - ratio| < 1e-6,
  (ii)  race near-tie     relative gap of the two smallest keys < 1e-6,
  (iii) ill-conditioned residual  r(x) / max(p, q) < 1e-6 at the winner.
Any other difference in a sampled decision is a failure. Trials whose rows
all agree must agree bit for bit in every output (meta, committed tokens,
next window)."""
import numpy as np

TIE = 1e-6


def compare_verify(gpu, ref, *, K, D, report=None):
    """gpu/ref: dicts of numpy arrays with keys meta, tok, next, sib, rows;
    ref also has margin. Returns (n_rows_mismatch, n_explained)."""
    B, L = ref["tok"].shape
    row_bad = np.zeros((B, L), bool)
    explained = 0
    unexplained = []
    gr, rr, mg = gpu["rows"], ref["rows"], ref["margin"]
    diff = (gr != rr).any(-1)
    for b, j in zip(*np.nonzero(diff)):
        m = mg[b, j]
        if m[0] < TIE or m[1] < TIE or m[3] < TIE:
            explained += 1
            row_bad[b, j] = True
        else:
            unexplained.append((int(b), int(j), gr[b, j].tolist(), rr[b, j].tolist(), m.tolist()))
    assert not unexplained, f"unexplained row mismatches (b, j, gpu, oracle, margins): {unexplained[:10]}"
    trial_ok = ~row_bad.any(1)
    for key in ("meta", "tok", "next"):
        g, r = gpu[key][trial_ok], ref[key][trial_ok]
        bad = np.nonzero((g != r).reshape(g.shape[0], -1).any(1))[0]
        assert bad.size == 0, f"{key} differs on trials {np.nonzero(trial_ok)[0][bad][:10]}"
    if D > 0 and K > 1:
        g, r = gpu["sib"][trial_ok], ref["sib"][trial_ok]
        ids = np.nonzero(trial_ok)[0]
        for t in np.nonzero((g != r).reshape(g.shape[0], -1).any(1))[0]:
            b = ids[t]
            n_c = ref["meta"][b, 0]
            Dn = ref["meta"][b, 2]
            gaps = [mg[b, n_c + d, 2] for d in range(Dn)]
            assert min(gaps) < TIE, f"sibling draw differs on trial {b} without a near-tie"
            explained += 1
    if report is not None:
        report.append(dict(rows_mismatch=int(diff.sum()), explained=explained, trials=B))
    return int(diff.sum()), explained
