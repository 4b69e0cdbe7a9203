"""GPU parity of sjd_verify (HIP, through the C ABI) with the oracle on the
same seeded inputs: token indices, stages and accepted lengths bit-exact
(decisions within 1e-6 of a tie are reported instead), probabilities within
1e-5 absolute."""
import numpy as np
import pytest
import torch

from oracle.parity import compare_verify
from synth_inputs import CONFIGS, verify_inputs

pytestmark = pytest.mark.gpu


def run_both(orc, inp, *, K, D, top_k, T=1.0, flags=3, seed=1, step=0, vis_lo=0, eol=-1, row_len=0,
             want_p=True, oracle_trials=None, gpu_flags=0):
    import paper_2603_18599_amd as sjd
    from paper_2603_18599_amd.sjd import verify_outputs
    dev = {k: (v.cuda() if v is not None else None) for k, v in inp.items()}
    B, L, V = dev["cur"].shape
    out = verify_outputs(B, L, K, D)
    rows = torch.zeros(B, L, 2, dtype=torch.int32, device="cuda")
    dbg = torch.zeros(B, L, V, dtype=torch.float32, device="cuda") if want_p else None
    sjd.sjd_verify(dev["cur"], dev["draft"], dev["draft_tok"], dev["meta"], out, K=K, D=D, top_k=top_k,
                   temperature=T, flags=flags | gpu_flags, seed=seed, step=step, sib=dev["sib"], vis_lo=vis_lo,
                   eol_id=eol,
                   row_len=row_len, out_rows=rows, dbg_p=dbg)
    torch.cuda.synchronize()
    idx = np.arange(B) if oracle_trials is None else np.asarray(oracle_trials)
    cpu = {k: (v[idx].numpy() if v is not None else None) for k, v in inp.items()}
    # trial index is a counter word: keep each trial's own index for the oracle
    if oracle_trials is None:
        ref = orc.verify(cpu["cur"], cpu["draft"], cpu["draft_tok"], cpu["meta"], K=K, D=D, top_k=top_k, T=T,
                         flags=flags, seed=seed, step=step, sib=cpu["sib"], vis_lo=vis_lo, eol_id=eol,
                         row_len=row_len, want_p=want_p)
    else:
        ref = orc_verify_trials(orc, cpu, idx, K=K, D=D, top_k=top_k, T=T, flags=flags, seed=seed, step=step,
                                vis_lo=vis_lo, eol=eol, row_len=row_len, want_p=want_p)
    gpu = dict(meta=out["meta"].cpu().numpy()[idx], tok=out["tok"].cpu().numpy()[idx],
               next=out["next"].cpu().numpy()[idx], sib=out["sib"].cpu().numpy()[idx],
               rows=rows.cpu().numpy()[idx])
    if want_p:
        gpu["p"] = dbg.cpu().numpy()[idx]
    return gpu, ref


def orc_verify_trials(orc, sub, trial_ids, **kw):
    """Oracle on a subset of trials, each at its own trial index (counter
    word 1), one call per trial."""
    outs = []
    for t, b in enumerate(trial_ids):
        one = {k: (v[t:t + 1] if v is not None else None) for k, v in sub.items()}
        r = orc.verify(one["cur"], one["draft"], one["draft_tok"], one["meta"], K=kw["K"], D=kw["D"],
                       top_k=kw["top_k"], T=kw["T"], flags=kw["flags"], seed=kw["seed"], step=kw["step"],
                       sib=one["sib"], vis_lo=kw["vis_lo"], eol_id=kw["eol"], row_len=kw["row_len"],
                       want_p=kw["want_p"], trial0=int(b))
        outs.append(r)
    return {k: np.concatenate([o[k] for o in outs]) for k in outs[0]}


def check(gpu, ref, K, D, want_p=True, label=None):
    import os
    if want_p:
        assert np.abs(gpu["p"] - ref["p"]).max() <= 1e-5
    return compare_verify(gpu, ref, K=K, D=D, label=label or os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0])


@pytest.mark.parametrize("V,top_k", [(1024, 0), (4096, 200), (16384, 2000), (65536, 2000)])
def test_verify_chain_matches_oracle(orc, V, top_k):
    B, L = 6, 32
    inp = verify_inputs(B, L, V, top_k=top_k, seed=V + top_k)
    gpu, ref = run_both(orc, inp, K=4, D=3, top_k=top_k, seed=7, step=3)
    check(gpu, ref, 4, 3)
    assert (gpu["meta"][:, 0] >= 1).all()


@pytest.mark.parametrize("V,top_k,T", [(4096, 200, 0.7), (16384, 2000, 1.9), (16384, 1500, 0.25), (2048, 0, 3.0), (65536, 2000, 0.6)])
def test_verify_temperature_matches_oracle(orc, V, top_k, T):
    # T != 1 divides every logit difference by T (T = 1 skips the division,
    # which returns its operand exactly); the tree rows exercise Theorem 2's
    # stages at the tempered distributions
    B, L, K, D = 4, 32, 4, 3
    inp = verify_inputs(B, L, V, top_k=top_k, seed=V + 17, K=K, D=D, D_in=2, draft_noise=1.0, temperature=T)
    gpu, ref = run_both(orc, inp, K=K, D=D, top_k=top_k, T=T, seed=13, step=2)
    check(gpu, ref, K, D)


@pytest.mark.parametrize("V,top_k", [(4096, 200), (16384, 2000), (32768, 2048)])
def test_verify_full_select_mode_matches_oracle(orc, V, top_k):
    """SJD_FULL_SELECT, the reference mode of the top-k selection (histograms
    over every row instead of the candidates at or above a sampled
    threshold), against the oracle: tree rows, drafting, residual draws."""
    from paper_2603_18599_amd.sjd import SJD_FULL_SELECT
    B, L, K, D = 6, 32, 4, 3
    inp = verify_inputs(B, L, V, top_k=top_k, seed=V + 5, K=K, D=D, D_in=2, draft_noise=1.0)
    gpu, ref = run_both(orc, inp, K=K, D=D, top_k=top_k, seed=21, step=1, gpu_flags=SJD_FULL_SELECT)
    check(gpu, ref, K, D)


def test_verify_selection_edge_rows(orc):
    """Rows whose top-k set the sampled threshold estimate handles badly or
    not at all, against the oracle (whichever selection the kernel takes):
    -inf entries (a few, or a third of the row); the kept set concentrated in
    one stripe of the row (every 2048 entries, the first 256 lifted by 4);
    logits on a coarse grid (long runs of equal values at the threshold, in
    the target and the draft row); a kept set of half and of nearly all of
    the row."""
    B, L, K, D = 8, 32, 4, 3
    V, top_k = 16384, 2000
    inp = verify_inputs(B, L, V, top_k=top_k, seed=77, K=K, D=D, D_in=2, draft_noise=1.0)
    g = torch.Generator().manual_seed(78)
    cur, dr = inp["cur"], inp["draft"]
    idx = torch.arange(V)
    for j in range(0, L, 4):
        few = torch.randint(0, V, (3,), generator=g)
        cur[0, j, few] = -float("inf")
        dr[1, j, few] = -float("inf")
    third = torch.rand(L, V, generator=g) < 0.33
    cur[2][third] = -float("inf")
    dr[2][torch.roll(third, 1, 1)] = -float("inf")
    stripe = (idx // 256) % 8 == 0
    cur[3][:, stripe] += 4.0
    dr[3][:, stripe] += 4.0
    cur[4] = torch.round(cur[4] * 2) / 2
    dr[4] = torch.round(dr[4] * 2) / 2
    cur[5] = torch.round(cur[5] * 8) / 8
    dr[5] = cur[5] + torch.round(torch.randn(L, V, generator=g) * 4) / 8
    # drafts must stay inside each draft row's kept set for the comparison to
    # exercise acceptances: redraw the spine drafts of the edited trials
    for b in range(6):
        vals, ix = torch.topk(dr[b], top_k, dim=1)
        pick = torch.multinomial(torch.softmax(vals.double(), 1), K, replacement=False, generator=g)
        toks = torch.gather(ix, 1, pick).to(torch.int32)
        inp["draft_tok"][b] = toks[:, 0]
        inp["sib"][b, :2] = toks[:2, 1:]
    gpu, ref = run_both(orc, inp, K=K, D=D, top_k=top_k, seed=5, step=2)
    check(gpu, ref, K, D)
    for V2, k2 in [(4096, 2048), (2048, 2000)]:
        inp2 = verify_inputs(4, L, V2, top_k=k2, seed=V2 + k2, K=K, D=D, D_in=1, draft_noise=1.0)
        gpu, ref = run_both(orc, inp2, K=K, D=D, top_k=k2, seed=6, step=3)
        check(gpu, ref, K, D)


def test_verify_tree_rows_with_siblings(orc):
    B, L, V, K, D = 8, 32, 4096, 4, 3
    inp = verify_inputs(B, L, V, top_k=300, seed=11, K=K, D=D, D_in=3, draft_noise=1.5)
    gpu, ref = run_both(orc, inp, K=K, D=D, top_k=300, seed=3, step=9)
    check(gpu, ref, K, D)
    # some sibling must have been tried somewhere
    assert (ref["rows"][:, :3, 1] != 1).any()


@pytest.mark.parametrize("V,top_k", [(4096, 300), (16384, 2000), (32768, 1000), (65536, 2000)])
@pytest.mark.parametrize("B", [8, 17])
def test_verify_drafting_in_row_kernel_and_after_finalize(orc, B, V, top_k):
    # launches of at most 512 rows draw the drafting candidates in the row
    # kernel, larger ones in a kernel of their own after finalize (from the
    # statistics the rows leave): both must match the oracle, at every
    # vocabulary tier
    L, K, D = 32, 4, 3
    inp = verify_inputs(B, L, V, top_k=top_k, seed=B * 7 + V, K=K, D=D, D_in=3, draft_noise=1.2)
    gpu, ref = run_both(orc, inp, K=K, D=D, top_k=top_k, seed=17, step=4, want_p=False)
    check(gpu, ref, K, D, want_p=False)
    assert (ref["sib"] >= 0).any()


def test_verify_placeholders_and_row_ends(orc):
    B, L, V = 6, 16, 2048
    inp = verify_inputs(B, L, V, top_k=100, seed=5, n_q=9)
    inp["meta"][:, 2] = torch.tensor([0, 3, 7, 10, 15, 44], dtype=torch.int32)
    eol = 5000
    W = 4
    for b in range(B):
        for j in range(L):
            if (int(inp["meta"][b, 2]) + j) % (W + 1) == W:
                inp["draft_tok"][b, j] = eol
    gpu, ref = run_both(orc, inp, K=4, D=3, top_k=100, seed=2, step=1, eol=eol, row_len=W, vis_lo=0)
    check(gpu, ref, 4, 3)


def test_verify_vanilla_sjd_mode(orc):
    B, L, V = 6, 32, 4096
    inp = verify_inputs(B, L, V, top_k=500, seed=21, draft_noise=2.0, K=1, D=0)
    gpu, ref = run_both(orc, inp, K=1, D=0, top_k=500, flags=0, seed=4)
    check(gpu, ref, 1, 0)


def test_verify_ties_in_logits(orc):
    # integer-valued logits: many exact ties at the top-k threshold
    B, L, V = 4, 8, 1024
    inp = verify_inputs(B, L, V, top_k=37, seed=9, int_logits=True, K=4, D=2)
    gpu, ref = run_both(orc, inp, K=4, D=2, top_k=37, seed=8)
    check(gpu, ref, 4, 2)


def test_verify_small_shapes(orc):
    for (B, L, V, top_k, K, D) in [(1, 1, 4, 0, 1, 0), (3, 1, 64, 1, 4, 0), (2, 5, 8, 3, 2, 2), (2, 64, 256, 17, 8, 8),
                                   (2, 3, 2048, 0, 2, 1), (2, 4, 20000, 2048, 4, 1), (1, 2, 40000, 1, 1, 0)]:
        inp = verify_inputs(B, L, V, top_k=top_k, seed=B * 100 + L, K=K, D=D)
        gpu, ref = run_both(orc, inp, K=K, D=D, top_k=top_k, seed=1)
        check(gpu, ref, K, D)


def test_verify_vis_range_offset(orc):
    B, L, V = 3, 16, 2048
    inp = verify_inputs(B, L, V, top_k=64, seed=31)
    lo = 151854
    inp["draft_tok"] += lo
    gpu, ref = run_both(orc, inp, K=4, D=3, top_k=64, seed=6, vis_lo=lo, eol=lo - 1, row_len=7)
    check(gpu, ref, 4, 3)
    assert (gpu["tok"][gpu["tok"] >= 0] >= lo - 1).all()


def test_verify_full_size_sampled(orc):
    """The benchmark's verify workload (4096 trials x 32 rows x 16384, top-2000)
    in the launch the benchmark times; the oracle checks 12 sampled trials."""
    c = CONFIGS["verify"]
    inp = verify_inputs(c["B"], c["L"], c["V"], top_k=c["top_k"], seed=1234, device="cuda")
    inp = {k: (v.cpu() if v is not None else None) for k, v in inp.items()}
    sample = [0, 1, 77, 500, 1023, 1024, 2047, 2048, 3000, 4000, 4094, 4095]
    gpu, ref = run_both(orc, inp, K=c["K"], D=c["D"], top_k=c["top_k"], seed=99, step=5, want_p=False,
                        oracle_trials=sample)
    compare_verify(gpu, ref, K=c["K"], D=c["D"], label="full-size 4096x32x16384, 12 sampled trials")


def test_verify_full_size_accept_length_closed_form():
    """At the benchmark's full size (4096 chain windows x 32 rows x 16384,
    top-2000), the mean committed length over the windows and four step
    indices matches its closed form. A step commits the accepted prefix plus
    one token (at most L) and, given the logits, the rows are independent:
    E[n_c] = 1 + sum_{i=1}^{L-1} prod_{j<i} a_j per window. With the drafted
    tokens x_j fixed (every step reuses them, only the accept draws are
    fresh), a_j = min(1, p_j(x_j) / q_j(x_j)); averaged over drafts drawn
    from q_j, a_j = sum_x min(p_j, q_j) (one minus the total variation
    distance). The first is checked against the kernel's outcomes, the second
    against the first (the inputs' drafts follow q)."""
    import paper_2603_18599_amd as sjd
    from paper_2603_18599_amd.sjd import verify_outputs
    c = CONFIGS["verify"]
    B, L, V, k = c["B"], c["L"], c["V"], c["top_k"]
    inp = verify_inputs(B, L, V, top_k=k, seed=4321, device="cuda")

    def topk_softmax(x):
        vals, idx = torch.topk(x, k, dim=1)
        return torch.zeros_like(x).scatter_(1, idx, torch.softmax(vals.double(), dim=1).float())

    def expect(a):
        return 1.0 + torch.cumprod(a[:, :L - 1], dim=1).sum(1)
    given, over = [], []
    for w0 in range(0, B, 128):
        p = topk_softmax(inp["cur"][w0:w0 + 128].reshape(-1, V))
        q = topk_softmax(inp["draft"][w0:w0 + 128].reshape(-1, V))
        x = inp["draft_tok"][w0:w0 + 128].reshape(-1, 1).long()
        given.append(expect(torch.clamp(p.gather(1, x).double() / q.gather(1, x).double(), max=1.0).view(-1, L)))
        over.append(expect(torch.minimum(p, q).double().sum(1).view(-1, L)))
    given, over = torch.cat(given).cpu().numpy(), torch.cat(over).cpu().numpy()
    ncs = []
    for step in range(4):
        out = verify_outputs(B, L, c["K"], c["D"])
        sjd.sjd_verify(inp["cur"], inp["draft"], inp["draft_tok"], inp["meta"], out, K=c["K"], D=c["D"], top_k=k,
                       seed=17, step=step)
        torch.cuda.synchronize()
        ncs.append(out["meta"][:, 0].cpu().numpy().astype(float))
    nc = np.stack(ncs)  # [step][window]
    se = nc.std() / np.sqrt(nc.size)
    d = given - over
    se_d = d.std() / np.sqrt(d.size)
    print(f"mean n_c {nc.mean():.4f}; closed form given the drafts {given.mean():.4f} (se {se:.4f}), "
          f"over draft draws {over.mean():.4f} (se {se_d:.4f})")
    assert abs(nc.mean() - given.mean()) < 5 * se
    assert abs(d.mean()) < 5 * se_d


def test_verify_is_deterministic(orc):
    import paper_2603_18599_amd as sjd
    from paper_2603_18599_amd.sjd import verify_outputs
    B, L, V = 64, 32, 16384
    inp = {k: (v.cuda() if v is not None else None) for k, v in verify_inputs(B, L, V, top_k=2000, seed=3).items()}
    res = []
    for _ in range(2):
        out = verify_outputs(B, L, 4, 3)
        sjd.sjd_verify(inp["cur"], inp["draft"], inp["draft_tok"], inp["meta"], out, K=4, D=3, top_k=2000, seed=5)
        torch.cuda.synchronize()
        res.append({k: v.cpu() for k, v in out.items()})
    for k in res[0]:
        assert torch.equal(res[0][k], res[1][k])


def test_verify_rejects_bad_arguments():
    import paper_2603_18599_amd as sjd
    from paper_2603_18599_amd.sjd import SjdError, verify_outputs
    inp = {k: (v.cuda() if v is not None else None) for k, v in verify_inputs(2, 4, 64, top_k=0, seed=1).items()}
    out = verify_outputs(2, 4, 4, 1)
    for kw in [dict(K=4, D=2), dict(K=9, D=0), dict(K=4, D=1, temperature=0.0), dict(K=4, D=1, top_k=-1)]:
        args = dict(K=4, D=1, top_k=0)
        args.update(kw)
        with pytest.raises(SjdError):
            sjd.sjd_verify(inp["cur"], inp["draft"], inp["draft_tok"], inp["meta"], out, **args)
