"""Comparison of sjd_verify (HIP) outputs with the oracle's (test
infrastructure: used by the GPU tests, the smoke check and the benchmark's
CPU-baseline leg), with the near-tie
classes of the parity bar:
  (i)   accept near-tie   |u - ratio| < 1e-6,
  (ii)  race near-tie     relative gap of the two smallest keys < 1e-6,
  (iii) ill-conditioned residual  r(x) / max(p, q) < 1e-6 at the winner,
  (iv)  drafting near-tie relative gap of consecutive drafting keys < 1e-6.
Any other difference in a sampled decision is a failure. Trials whose rows
all agree must agree bit for bit in every output (meta, committed tokens,
next window).

Every comparison is reported: how many decisions the oracle took within the
tie band of each class, and how many of the differing rows each class
explains. The records accumulate in RECORDS (printed at the end of the
pytest session by conftest.py)."""
import numpy as np

TIE = 1e-6
CLASSES = ("accept", "race", "drafting", "residual")  # oracle margin columns 0..3
RECORDS = []


def compare_verify(gpu, ref, *, K, D, report=None, label=""):
    """gpu/ref: dicts of numpy arrays with keys meta, tok, next, sib, rows;
    ref also has margin. Returns (n_rows_mismatch, n_explained); appends a
    record with the per-class counts to RECORDS (and to report, if given)."""
    B, L = ref["tok"].shape
    row_bad = np.zeros((B, L), bool)
    explained = 0
    expl_by = {c: 0 for c in CLASSES}
    unexplained = []
    gr, rr, mg = gpu["rows"], ref["rows"], ref["margin"]
    diff = (gr != rr).any(-1)
    for b, j in zip(*np.nonzero(diff)):
        m = mg[b, j]
        if m[0] < TIE or m[1] < TIE or m[3] < TIE:
            explained += 1
            row_bad[b, j] = True
            expl_by[CLASSES[int(np.argmin([m[0], m[1], np.inf, m[3]]))]] += 1
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
            expl_by["drafting"] += 1
    near = {c: int((mg[..., i] < TIE).sum()) for i, c in enumerate(CLASSES)}
    rec = dict(label=label, trials=int(B), rows=int(B * L), rows_mismatch=int(diff.sum()), explained=explained,
               near_ties=near, explained_by=expl_by)
    RECORDS.append(rec)
    if report is not None:
        report.append(rec)
    return int(diff.sum()), explained


def summary():
    """One line per comparison plus the totals."""
    if not RECORDS:
        return []
    lines = []
    tot = {c: 0 for c in CLASSES}
    tex = {c: 0 for c in CLASSES}
    rows = mism = 0
    for r in RECORDS:
        rows += r["rows"]
        mism += r["rows_mismatch"]
        for c in CLASSES:
            tot[c] += r["near_ties"][c]
            tex[c] += r["explained_by"][c]
        lines.append(f"{r['label'] or 'verify'}: {r['rows']} rows, {r['rows_mismatch']} differ "
                     f"(explained: {r['explained_by']}); decisions within 1e-6 of a tie: {r['near_ties']}")
    lines.append(f"total: {len(RECORDS)} comparisons, {rows} rows, {mism} rows differ, all explained "
                 f"(by class {tex}); near-tie decisions by class {tot}")
    return lines
