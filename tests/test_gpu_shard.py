"""GPU parity of the vocabulary-sharded calls (dsde_shard_*) against the CPU
oracle on the whole rows.

The G shards run on one GPU one after another (paper_2509_01083_amd.
verify_sharded); the exchanges are the stacked per-shard outputs.  The oracle
sees the unsplit rows, so these tests check that the split statistics, the
fold across slices, the slice-level inverse-CDF search and the in-slice draw
reproduce dsde_verify's results under the same comparison rules (bit-exact
outside the tie bands, KLD within tolerance).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.parity import KLD_ABS, KLD_REL, compare_verify
from tests.test_gpu_verify import announce, random_arrays, step_from_arrays

pytestmark = pytest.mark.gpu


def run_sharded(dsde, step, slices, row_lse=True):
    lse = torch.empty((max(step.N, 1), 2), dtype=torch.float64, device=step.target.device)[:step.N] \
        if row_lse else None
    out = dsde.verify_sharded(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                              step.u_acc, step.u_res, step.k_max, slices, row_lse=lse, draft_entropy=True)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items() if isinstance(v, torch.Tensor)}
    if lse is not None:
        res["row_lse"] = lse.cpu().numpy()
    return res


def check_sharded(dsde, step, slices, label):
    announce(f"{label}: B={step.B} N={step.N} V={step.V} dtype={step.target.dtype} slices={len(slices)}")
    got = run_sharded(dsde, step, slices)
    host = W.host_arrays(step)
    ref = oracle.verify(**host, n_threads=16)
    rep = compare_verify(got, ref, host["sl"], host["cu_sl"], label, host=host)
    # the all-reduced drawn token is the one written into tokens wherever a
    # token was drawn (no error): every drawing shard agrees with the owner
    fine = got["seq_err"] == 0
    idx = np.arange(step.B)
    drawn_tok = got["tokens"][idx, got["accepted"]]
    assert (got["drawn"][fine] == drawn_tok[fine]).all(), label
    assert (got["drawn"][~fine] == -1).all(), label
    print(f"[report] {label}: {rep}", flush=True)
    return got, ref, rep


@pytest.mark.parametrize("name", ["tiny", "b64", "greedy", "b256", "b256g"])
@pytest.mark.parametrize("G", [1, 2, 3, 8])
def test_workload_parity_sharded(gpu_lib, name, G):
    import paper_2509_01083_amd as dsde
    cfg = W.CONFIGS[name]
    step = W.make_step(cfg, seed=13, device="cuda")
    slices = dsde.slice_bounds(step.V, G)
    _, _, rep = check_sharded(dsde, step, slices, f"{name} over {len(slices)} slices")
    assert rep["compared"] >= 0.9 * step.B


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_ragged_and_unaligned_slices(gpu_lib, dtype):
    """Slices of widths that are not multiples of the vector width (the scalar
    row path), a slice narrower than one sub-block, and one wider than a chunk."""
    import paper_2509_01083_amd as dsde
    rng = np.random.default_rng(21)
    V = 20011
    sls = [3, 0, 1, 5, 2, 4, 1, 2]
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    step = step_from_arrays(target, draft, sls, tokens, [1.0, 0.7] * 4, u_acc, u_res, 5, dtype)
    slices = [(0, 5000), (5000, 5003), (5003, 5300), (5300, 16000), (16000, V)]
    check_sharded(dsde, step, slices, f"ragged slices {dtype}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_sharded_draw_at_slice_and_chunk_boundaries(gpu_lib, dtype):
    """All draw mass on tokens at the edges of slices, chunks and sub-blocks,
    u' in the middle of each token's CDF interval: rejected sequences draw from
    the residual, accepted ones from the bonus row, each landing on a known
    token in a known slice."""
    import paper_2509_01083_amd as dsde
    V = 3 * 8192 + 704
    hot = np.array([0, 511, 512, 8191, 8192, 12287, 12288, 16383, 16384, 24575, 24576, V - 1])
    slices = [(0, 8192), (8192, 12288), (12288, 16384), (16384, V)]
    H = len(hot)
    B = 2 * H
    sls = [1] * B
    rng = np.random.default_rng(V)
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    other = 3000
    for b in range(B):
        row = np.full(V, -30.0, np.float32)
        row[hot] = 0.0
        if b < H:
            target[2 * b] = row
            draft[b] = -30.0
            draft[b, other] = 30.0
            u_acc[b] = 0.5
        else:
            draft[b] = target[2 * b]
            u_acc[b] = 0.0
            target[2 * b + 1] = row
        tokens[b] = other
        u_res[b] = (b % H + 0.5) / H
    step = step_from_arrays(target, draft, sls, tokens, [1.0] * B, u_acc, u_res, 1, dtype)
    got, _, rep = check_sharded(dsde, step, slices, f"sharded draw at boundaries {dtype}")
    assert rep["compared"] == B, rep
    assert (got["accepted"] == np.array([0] * H + [1] * H)).all()
    assert (got["tokens"][np.arange(B), got["accepted"]] == np.concatenate([hot, hot])).all()


def test_sharded_error_contract(gpu_lib):
    """The error bits and fallbacks of dsde_verify, with the offending values in
    different slices."""
    import paper_2509_01083_amd as dsde
    rng = np.random.default_rng(6)
    sls = [2, 2, 2, 2, 2, 2, 2]
    V = 9000
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    temps = np.ones(7, np.float32)
    tokens[2] = V                  # seq 1: token out of range
    u_acc[4] = 1.0                 # seq 2: uniform out of [0, 1)
    temps[3] = 2.0 ** 17           # seq 3: temperature out of range
    draft[8, 17] = np.nan          # seq 4: NaN in a drafted pair (slice 0)
    target[5 * 3 + 1, 8000] = -np.inf  # seq 5: -inf in a drafted target row (last slice)
    target[6 * 3: 6 * 3 + 2] = draft[12:14]  # seq 6: both accepted, bonus row has +inf (middle slice)
    u_acc[12:14] = 0.99999
    target[6 * 3 + 2, 4500] = np.inf
    step = step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, 2)
    got, _, _ = check_sharded(dsde, step, dsde.slice_bounds(V, 3), "sharded error contract")
    assert list(got["seq_err"]) == [0, 2, 16, 8, 4, 4, 4]
    assert np.isnan(got["kld"][2:12]).all() and np.isfinite(got["kld"][:2]).all()
    assert np.isfinite(got["kld"][12:14]).all()


def test_token_in_no_slice_or_two_is_an_error(gpu_lib):
    """Slices that leave a gap or overlap: a drafted token no slice holds, or two
    slices hold, flags its sequence (DSDE_ERR_TOKEN)."""
    import paper_2509_01083_amd as dsde
    rng = np.random.default_rng(8)
    sls = [1, 1, 1]
    V = 1000
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    tokens[:] = [100, 750, 900]
    step = step_from_arrays(target, draft, sls, tokens, [1.0] * 3, u_acc, u_res, 1)
    announce("token ownership")
    out = dsde.verify_sharded(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                              step.u_acc, step.u_res, 1, [(0, 400), (350, 700), (800, 1000)])
    err = out["seq_err"].cpu().numpy()
    assert err[0] == 0 and err[2] == 0 and err[1] & 2, err  # 750 lies in no slice
    out = dsde.verify_sharded(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                              step.u_acc, step.u_res, 1, [(0, 400), (50, 1000)])
    err = out["seq_err"].cpu().numpy()
    assert err[0] & 2 and err[1] == 0 and err[2] == 0, err  # 100 lies in both


def test_sharded_equals_unsharded_on_kld(gpu_lib):
    """dsde_verify and the sharded calls on the same b256 step: identical error
    bits, and KLD values that differ only by the rounding of the split sums."""
    import paper_2509_01083_amd as dsde
    from tests.parity import run_verify
    step = W.make_step(W.CONFIGS["b256"], seed=3, device="cuda")
    announce("sharded vs unsharded b256")
    whole = run_verify(dsde, step)
    split = run_sharded(dsde, step, dsde.slice_bounds(step.V, 8))
    assert np.array_equal(whole["seq_err"], split["seq_err"])
    d = np.abs(whole["kld"].astype(np.float64) - split["kld"].astype(np.float64))
    assert (d <= KLD_REL * np.abs(whole["kld"]) + KLD_ABS).all(), d.max()


@pytest.mark.parametrize("name", ["b256", "greedy", "layout"])
def test_fused_shard_acceptance_equals_the_three_calls(gpu_lib, name):
    """dsde_shard_accept_step against dsde_shard_accept, dsde_kld_signal and
    dsde_next_sl in turn, from the same gathered partials: identical bits (the
    layout case breaks cu_sl: every sequence flagged, the SL rule still runs)."""
    import paper_2509_01083_amd as dsde
    cfg = W.CONFIGS["b64" if name == "layout" else name]
    step = W.make_step(cfg, seed=17, device="cuda")
    if name == "layout":
        cu = step.cu_sl.clone()
        cu[1] += 1
        step = W.Step(**{**step.__dict__, "cu_sl": cu})
    announce(f"fused shard acceptance {name}")
    base = dsde.verify_sharded(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                               step.u_acc, step.u_res, step.k_max, dsde.slice_bounds(step.V, 4))
    parts, err0 = base["parts"], base["shard_seq_err"][0]
    st = W.make_signal_state(cfg, seed=17, device="cuda")
    st_a = W.SignalState(hist=st.hist.clone(), head=st.head.clone(), count=st.count.clone(), sl_max=st.sl_max)
    st_b = W.SignalState(hist=st.hist.clone(), head=st.head.clone(), count=st.count.clone(), sl_max=st.sl_max)
    budget = torch.as_tensor(np.random.default_rng(5).integers(0, 10, step.B).astype(np.int32), device="cuda")
    args = (parts, step.V, step.sl, step.cu_sl, step.draft_tokens, step.temperature, step.u_acc, step.u_res,
            step.k_max)
    e_a = err0.clone()
    a = dsde.shard_accept(*args, e_a, draft_entropy=True)
    s_ = dsde.kld_signal(step.sl, step.cu_sl, a["kld"], st_a.hist, st_a.head, st_a.count)
    n_ = dsde.next_sl(s_["sf"], s_["wvir"], st_a.sl_max, 2.0, step.k_max, budget=budget)
    e_b = err0.clone()
    f = dsde.shard_accept_step(*args, e_b, st_b.hist, st_b.head, st_b.count, st_b.sl_max, draft_entropy=True,
                               budget=budget)
    torch.cuda.synchronize()
    chain = {**a, **s_, **n_}
    for k in ("accepted", "tokens", "jobs", "sl_next"):
        assert torch.equal(chain[k], f[k]), k
    written = ("mu_last", "var_short", "var_long", "wvir", "sf", "sl_hat", "sl_cap")
    if name != "layout":  # the KLD is not written under an invalid layout
        written = ("kld", "draft_entropy") + written
    for k in written:
        assert torch.equal(chain[k].view(torch.int32), f[k].view(torch.int32)), k
    assert torch.equal(st_a.hist.view(torch.int32), st_b.hist.view(torch.int32))
    assert torch.equal(st_a.head, st_b.head) and torch.equal(st_a.count, st_b.count)
    assert torch.equal(e_a | s_["seq_err"] | n_["seq_err"], e_b)
    if name == "layout":
        assert (e_b.cpu().numpy() & 1).all()
