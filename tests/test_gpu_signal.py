"""GPU parity of dsde_kld_signal and dsde_next_sl against the CPU oracle, alone
and chained behind dsde_verify (including the multi-step controller loop).

Tolerances: mu_last, SF, WVIR, SL_hat and the cap within 1e-4 relative;
variances within 1e-4 relative plus 1e-9 absolute.  SL decisions are
bit-exact except where the oracle's tie analysis flags them: in isolation
(identical float inputs) only decisions within 1e-5 of a rounding boundary;
behind dsde_verify, also decisions that a relative change of 1e-4 in any KLD
history entry (the KLD tolerance) could flip.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.helpers import packed_layout
from tests.parity import compare_verify, run_verify

pytestmark = pytest.mark.gpu

REL = 1e-4


def announce(msg):
    print(f"\n[case] {msg}", flush=True)


def close(got, ref, rel=REL, abs_=0.0, label=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = ~(np.abs(got - ref) <= rel * np.abs(ref) + abs_)
    bad &= ~(np.isnan(got) & np.isnan(ref))
    assert not bad.any(), f"{label}: {np.nonzero(bad)[0][:8]} got {got[bad][:4]} ref {ref[bad][:4]}"


def gpu_signal(dsde, sl, cu, kld, st, n_short=10, n_long=30, delta=0.85, eps=1e-6):
    out = dsde.kld_signal(sl, cu, kld, st.hist, st.head, st.count, n_short, n_long, delta, eps)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def compare_signal(got, ref, label, spread=None):
    """Signal outputs within 1e-4 relative (variances + 1e-9 absolute), widened by the
    oracle's first-order spread when the inputs themselves differ within the KLD
    tolerance (chained comparisons)."""
    assert np.array_equal(got["seq_err"].astype(np.uint32), ref["seq_err"]), label
    zero = np.zeros_like(ref["mu_last"])
    sp = spread or {}
    close(got["mu_last"], ref["mu_last"], abs_=0.0, label=f"{label} mu_last")
    for k, floor in (("sf", 0.0), ("wvir", 0.0), ("var_short", 1e-9), ("var_long", 1e-9)):
        extra = np.nan_to_num(sp.get("d_" + k, zero))
        got_k = np.asarray(got[k], np.float64)
        ref_k = np.asarray(ref[k], np.float64)
        bad = ~(np.abs(got_k - ref_k) <= REL * np.abs(ref_k) + floor + extra)
        bad &= ~(np.isnan(got_k) & np.isnan(ref_k))
        assert not bad.any(), f"{label} {k}: {np.nonzero(bad)[0][:8]} got {got_k[bad][:4]} ref {ref_k[bad][:4]}"


@pytest.mark.parametrize("W_, n_short, n_long", [(32, 10, 30), (8, 10, 30), (16, 3, 12), (40, 10, 30)])
def test_kld_signal_alone(gpu_lib, W_, n_short, n_long):
    announce(f"kld_signal W={W_} windows={n_short}/{n_long}")
    rng = np.random.default_rng(W_)
    B = 300
    sls = rng.integers(0, 9, B)
    sl, cu = packed_layout(sls)
    kld = (rng.gamma(0.6, 0.5, int(cu[-1]))).astype(np.float32)
    cfg = dict(W.CONFIGS["b256"], B=B, W=W_)
    st = W.make_signal_state(cfg, seed=3, device="cuda")
    # a few partly filled and empty rings
    cnt = st.count.cpu().numpy()
    cnt[::7] = rng.integers(0, W_ + 1, len(cnt[::7]))
    cnt[5] = 0
    st.count.copy_(torch.as_tensor(cnt))
    h0, hd0, c0 = st.hist.cpu().numpy(), st.head.cpu().numpy(), st.count.cpu().numpy()
    dev = lambda x: torch.as_tensor(x, device="cuda")
    got = gpu_signal(gpu_lib, dev(sl), dev(cu), dev(kld), st, n_short, n_long)
    ref = oracle.kld_signal(sl, cu, kld.astype(np.float64), h0, hd0, c0, n_short, n_long)
    compare_signal(got, ref, "signal")
    assert np.array_equal(st.head.cpu().numpy(), ref["head"])
    assert np.array_equal(st.count.cpu().numpy(), ref["count"])
    close(st.hist.cpu().numpy(), ref["hist"], rel=1e-7, label="ring")


def test_kld_signal_errors(gpu_lib):
    announce("kld_signal errors")
    sls = [2, 0, 3, 1]
    sl, cu = packed_layout(sls)
    kld = np.array([0.1, 0.2, np.nan, 0.3, 0.4, 0.5], np.float32)
    cfg = dict(W.CONFIGS["b64"], B=4)
    st = W.make_signal_state(cfg, seed=1, device="cuda")
    st.head[3] = 99  # bad ring state
    h0, hd0, c0 = st.hist.cpu().numpy(), st.head.cpu().numpy(), st.count.cpu().numpy()
    dev = lambda x: torch.as_tensor(x, device="cuda")
    got = gpu_signal(gpu_lib, dev(sl), dev(cu), dev(kld), st)
    ref = oracle.kld_signal(sl, cu, kld.astype(np.float64), h0, hd0, c0)
    assert list(got["seq_err"]) == [0, 0, 32, 64]
    compare_signal(got, ref, "signal errors")
    cu_bad = cu.copy()
    cu_bad[2] += 1
    got = gpu_signal(gpu_lib, dev(sl), dev(cu_bad), dev(kld), st)
    assert (got["seq_err"] == 1).all()


def sl_decision_ties(hat, cap, seq_err, sl_min, sl_hi, tau=1e-5):
    return oracle.sl_round_ties(hat, np.zeros_like(hat), seq_err, sl_min, sl_hi, tau)


def test_next_sl_alone(gpu_lib):
    announce("next_sl")
    rng = np.random.default_rng(9)
    B = 2000
    sf = (rng.gamma(0.5, 0.6, B)).astype(np.float32)
    wvir = (rng.gamma(1.0, 0.8, B)).astype(np.float32)
    sl_max = rng.choice([8.0, 16.0, 6.5], B).astype(np.float32)
    sf[7] = np.nan
    sl_max[11] = 1.0  # below sl_min
    dev = lambda x: torch.as_tensor(x, device="cuda")
    out = gpu_lib.next_sl(dev(sf), dev(wvir), dev(sl_max), 2.0, 16)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    ref = oracle.next_sl(sf.astype(np.float64), wvir.astype(np.float64), sl_max.astype(np.float64), 2.0, 16)
    assert np.array_equal(got["seq_err"].astype(np.uint32), ref["seq_err"])
    close(got["sl_hat"], ref["sl_hat"], label="sl_hat")
    close(got["sl_cap"], [ref["sl_cap"]], label="cap")
    ties = sl_decision_ties(ref["sl_hat"], ref["sl_cap"], ref["seq_err"], 2.0, 16)
    ok = ties == 0
    assert np.array_equal(got["sl_next"][ok], ref["sl_next"][ok])
    print(f"[report] next_sl ties={int(ties.sum())} of {B}", flush=True)
    # the per-sequence token budget (Sec. 3.2): min(SL_next, max(budget - 1, 0))
    budget = rng.integers(-2, 20, B).astype(np.int32)
    out_b = gpu_lib.next_sl(dev(sf), dev(wvir), dev(sl_max), 2.0, 16, budget=dev(budget))
    torch.cuda.synchronize()
    ref_b = oracle.next_sl(sf.astype(np.float64), wvir.astype(np.float64), sl_max.astype(np.float64), 2.0, 16,
                           budget=budget)
    nb = out_b["sl_next"].cpu().numpy()
    tight = budget - 1 <= 2  # the budget decides, whatever the rounding
    assert np.array_equal(nb[ok | tight], ref_b["sl_next"][ok | tight])
    assert np.array_equal(out_b["sl_cap"].cpu().numpy(), out["sl_cap"].cpu().numpy())


def oracle_chain(host, h0, hd0, c0, smax, sl_hi):
    ref = oracle.verify(**host, n_threads=16)
    sr = oracle.kld_signal(host["sl"], host["cu_sl"], ref["kld"], h0, hd0, c0)
    nr = oracle.next_sl(sr["sf"], sr["wvir"], smax, 2.0, sl_hi)
    spread = oracle.signal_spread(sr["hist"], sr["head"], sr["count"], smax, nr["seq_err"] | sr["seq_err"],
                                  rho=1e-4)
    return ref, sr, nr, spread


# Largest fraction of a batch's SL decisions that may fall in the tie band:
# SL_hat's first-order spread under the KLD tolerance is ~1e-4 per unit of
# SL, so a few decisions per thousand land within it of a rounding boundary.
MAX_SL_TIE_FRACTION = 0.02


def compare_sl(ng, nr, sr, spread, smax, sl_hi, label, max_tie_fraction=MAX_SL_TIE_FRACTION):
    """SL decisions bit-exact outside the tie band, and the band itself kept
    small: at most ``max_tie_fraction`` of the sequences without an error
    (None: checked by the caller over a whole run)."""
    assert np.array_equal(ng["seq_err"].astype(np.uint32) & 32, nr["seq_err"] & 32), label
    hat_tol = REL * np.abs(nr["sl_hat"]) + np.nan_to_num(spread["d_sl_hat"]) + 1e-6
    ok_hat = np.isnan(nr["sl_hat"]) | (np.abs(ng["sl_hat"] - nr["sl_hat"]) <= hat_tol)
    assert ok_hat.all(), f"{label} sl_hat: {np.nonzero(~ok_hat)[0][:8]}"
    ties = oracle.sl_round_ties(spread["sl_hat"], spread["d_sl_hat"], nr["seq_err"], 2.0, sl_hi, tau=1e-5)
    ok = ties == 0
    mism = np.nonzero(ok & (ng["sl_next"] != nr["sl_next"]))[0]
    assert mism.size == 0, f"{label}: SL decisions differ at {mism[:8]}"
    n_fine = int((nr["seq_err"] == 0).sum())
    n_ties = int(ties.sum())
    print(f"[report] {label}: SL decisions compared {n_fine - n_ties}, ties {n_ties}", flush=True)
    if max_tie_fraction is not None:
        assert n_ties <= max_tie_fraction * n_fine, f"{label}: {n_ties} SL ties of {n_fine}"
    return n_ties


def chained_step(dsde, step, st, sl_max, sl_hi, label, max_tie_fraction=MAX_SL_TIE_FRACTION):
    """verify -> kld_signal -> next_sl on the GPU and the oracle's chain; compares every stage."""
    h0, hd0, c0 = st.hist.cpu().numpy(), st.head.cpu().numpy(), st.count.cpu().numpy()
    got = run_verify(dsde, step, row_lse=False)
    host = W.host_arrays(step)
    smax = sl_max.cpu().numpy().astype(np.float64)
    ref, sr, nr, spread = oracle_chain(host, h0, hd0, c0, smax, sl_hi)
    rep = compare_verify(got, ref, host["sl"], host["cu_sl"], label, host=host)
    kld_t = torch.as_tensor(got["kld"], device="cuda")
    sg = gpu_signal(dsde, step.sl, step.cu_sl, kld_t, st)
    compare_signal(sg, sr, f"{label} signal", spread)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    out = dsde.next_sl(dev(sg["sf"]), dev(sg["wvir"]), sl_max, 2.0, sl_hi)
    torch.cuda.synchronize()
    ng = {k: v.cpu().numpy() for k, v in out.items()}
    rep["sl_ties"] = compare_sl(ng, nr, sr, spread, smax, sl_hi, label, max_tie_fraction)
    return ng, nr, sr, rep


@pytest.mark.parametrize("name", ["tiny", "b64", "b256", "lowacc", "spread"])
def test_chained_step(gpu_lib, name):
    cfg = W.CONFIGS[name]
    step = W.make_step(cfg, seed=21, device="cuda")
    st = W.make_signal_state(cfg, seed=21, device="cuda")
    announce(f"chained {name} B={step.B} N={step.N} V={step.V}")
    ng, nr, _, rep = chained_step(gpu_lib, step, st, st.sl_max, cfg.get("sl_hi", cfg["k_max"]), name)
    rep["sl_next_values"] = {int(v): int(c) for v, c in zip(*np.unique(ng["sl_next"], return_counts=True))}
    rep["sl_cap"] = float(nr["sl_cap"])
    print(f"[report] chained {name}: {rep}", flush=True)


@pytest.mark.parametrize("seed", [21, 22])
def test_chained_step_decisions_spread(gpu_lib, seed):
    """Close drafts and per-sequence SL_max in [4, 16]: small penalties, so
    Eqs. 2, 8 and 11 decide many different lengths and the cap sits far above
    SL_min.  At least four distinct next lengths must be compared bit-exactly,
    so a rule stuck at SL_min, or one that ignored SL_max, WVIR or the cap,
    could not pass."""
    cfg = W.CONFIGS["spread"]
    step = W.make_step(cfg, seed=seed, device="cuda")
    st = W.make_signal_state(cfg, seed=seed, device="cuda")
    announce(f"chained spread seed {seed} B={step.B} N={step.N}")
    ng, nr, sr, rep = chained_step(gpu_lib, step, st, st.sl_max, cfg["sl_hi"], f"spread {seed}")
    ok = nr["seq_err"] == 0
    values = np.unique(nr["sl_next"][ok])
    assert values.size >= 4, values
    assert nr["sl_cap"] > 4.0
    assert (ng["sl_next"][ok] >= 2).all() and (ng["sl_next"][ok] <= np.ceil(nr["sl_cap"])).all()
    below_cap = ok & (nr["sl_hat"] < nr["sl_cap"] - 0.5)  # decided by Eq. 2 / 8 alone, not by the cap
    assert np.unique(nr["sl_next"][below_cap]).size >= 3
    print(f"[report] spread {seed}: next lengths {values.tolist()}, cap {nr['sl_cap']:.3f}, "
          f"{int(below_cap.sum())} below the cap, ties {rep['sl_ties']}", flush=True)


def run_loop(dsde, cfg, steps, seed, label):
    """The multi-step controller: each step's SLs come from the previous step's
    decisions, with fresh seeded logits every step and the per-sequence draft
    noise on its random walk.  Both sides use the oracle's decisions to build
    the next step, so a tie can never fork the two trajectories; every stage
    of the GPU step is compared at every step.  The GPU's ring evolves on its
    own (the oracle keeps its own fp64 ring), so pushes, window sizes and the
    wrap-around of the GPU ring are checked as the run goes."""
    B = cfg["B"]
    st = W.make_signal_state(cfg, seed=seed, device="cuda")
    sl = W.sample_sl(cfg, seed)
    sigma = W.initial_sigma(cfg, seed)
    total_ties, total_cmp, distinct, kld_ratio = 0, 0, set(), 0.0
    h_or, hd_or, c_or = st.hist.cpu().numpy().astype(np.float64), st.head.cpu().numpy(), st.count.cpu().numpy()
    for t in range(steps):
        step = W.make_step(cfg, seed=seed, device="cuda", step=t, sl=sl, sigma=sigma)
        announce(f"{label} step {t}: N={step.N}")
        host = W.host_arrays(step)
        got = run_verify(dsde, step, row_lse=False)
        smax = st.sl_max.cpu().numpy().astype(np.float64)
        ref, sr, nr, spread = oracle_chain(host, h_or, hd_or, c_or, smax, cfg["k_max"])
        rep = compare_verify(got, ref, host["sl"], host["cu_sl"], f"{label} step {t}", host=host)
        kld_ratio = max(kld_ratio, rep.get("kld_err_over_tol", 0.0))
        sg = gpu_signal(dsde, step.sl, step.cu_sl, torch.as_tensor(got["kld"], device="cuda"), st)
        compare_signal(sg, sr, f"{label} step {t} signal", spread)
        assert np.array_equal(st.head.cpu().numpy(), sr["head"]) and np.array_equal(st.count.cpu().numpy(),
                                                                                     sr["count"])
        close(st.hist.cpu().numpy(), sr["hist"], rel=1e-4, abs_=1e-7, label=f"{label} step {t} ring")
        dev = lambda x: torch.as_tensor(x, device="cuda")
        out = dsde.next_sl(dev(sg["sf"]), dev(sg["wvir"]), st.sl_max, 2.0, cfg["k_max"])
        torch.cuda.synchronize()
        ng = {k: v.cpu().numpy() for k, v in out.items()}
        total_ties += compare_sl(ng, nr, sr, spread, smax, cfg["k_max"], f"{label} step {t}", None)
        total_cmp += int((nr["seq_err"] == 0).sum())
        distinct |= set(np.unique(nr["sl_next"]).tolist())
        h_or, hd_or, c_or = sr["hist"], sr["head"], sr["count"]
        sl = nr["sl_next"]
        sigma = W.walk_sigma(sigma, cfg, seed, t)
    print(f"[report] {label}: {steps} steps, SL ties {total_ties} of {total_cmp}, "
          f"next lengths seen {sorted(distinct)}, worst KLD error / tolerance {kld_ratio:.3f}", flush=True)
    assert total_ties <= MAX_SL_TIE_FRACTION * total_cmp
    if steps > cfg["W"]:
        assert (c_or == cfg["W"]).all()  # every ring filled and wrapped


def test_controller_loop_reduced_vocab(gpu_lib):
    cfg = dict(W.CONFIGS["loop"], B=256, V=4096)
    announce("controller loop B=256 V=4096 200 steps")
    run_loop(gpu_lib, cfg, 200, seed=5, label="loop-reduced")


@pytest.mark.timeout(900)
def test_controller_loop_full_shape(gpu_lib):
    """The controller loop at its stated shape (B = 1024, V = 128256, W = 32,
    empty rings at the start): 40 steps, so every ring fills after 32 steps
    and wraps for the last eight."""
    cfg = W.CONFIGS["loop"]
    announce("controller loop B=1024 V=128256 40 steps")
    run_loop(gpu_lib, cfg, 40, seed=6, label="loop-full")


def clone_state(st):
    return W.SignalState(hist=st.hist.clone(), head=st.head.clone(), count=st.count.clone(),
                         sl_max=st.sl_max.clone())


# more sequences than the set-up kernel and the cap kernel hold in registers
# (their looping paths), half of them greedy
WIDE = dict(W.CONFIGS["greedy"], B=1500, V=512)


@pytest.mark.parametrize("name", ["tiny", "b64", "b256", "greedy", "wide", "layout", "wide_layout"])
def test_fused_step_equals_the_three_calls(gpu_lib, name):
    """dsde_step against dsde_verify, dsde_kld_signal and dsde_next_sl in turn:
    identical bits.  The layout cases break cu_sl, which flags every sequence
    before any row is read; the SL rule still runs on the flagged batch."""
    cfg = WIDE if name.startswith("wide") else W.CONFIGS["b64" if name == "layout" else name]
    step = W.make_step(cfg, seed=31, device="cuda")
    if name.endswith("layout"):
        cu = step.cu_sl.clone()
        cu[1] += 1
        step = W.Step(**{**step.__dict__, "cu_sl": cu})
    st = W.make_signal_state(cfg, seed=31, device="cuda")
    announce(f"fused step vs chain {name}")
    st_a, st_b = clone_state(st), clone_state(st)
    budget = torch.as_tensor(np.random.default_rng(3).integers(0, 10, step.B).astype(np.int32), device="cuda")
    v = gpu_lib.verify(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                       step.u_acc, step.u_res, step.k_max, draft_entropy=True)
    s_ = gpu_lib.kld_signal(step.sl, step.cu_sl, v["kld"], st_a.hist, st_a.head, st_a.count)
    n_ = gpu_lib.next_sl(s_["sf"], s_["wvir"], st_a.sl_max, 2.0, step.k_max, budget=budget)
    f = gpu_lib.step(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                     step.u_acc, step.u_res, step.k_max, st_b.hist, st_b.head, st_b.count, st_b.sl_max,
                     draft_entropy=True, budget=budget)
    torch.cuda.synchronize()
    chain = {**v, **s_, **n_}
    for k in ("accepted", "tokens", "sl_next"):
        assert torch.equal(chain[k], f[k]), k
    written = ("mu_last", "var_short", "var_long", "wvir", "sf", "sl_hat", "sl_cap")
    if not name.endswith("layout"):  # the KLD is not written under an invalid layout
        written = ("kld", "draft_entropy") + written
    for k in written:
        assert torch.equal(chain[k].view(torch.int32), f[k].view(torch.int32)), k
    assert torch.equal(st_a.hist.view(torch.int32), st_b.hist.view(torch.int32))
    assert torch.equal(st_a.head, st_b.head) and torch.equal(st_a.count, st_b.count)
    assert torch.equal(v["seq_err"] | s_["seq_err"] | n_["seq_err"], f["seq_err"])
    if name.endswith("layout"):
        assert (f["seq_err"].cpu().numpy() & 1).all()


@pytest.mark.parametrize("name", ["b256", "lowacc", "b256g"])
def test_fused_step_parity(gpu_lib, name):
    cfg = W.CONFIGS[name]
    step = W.make_step(cfg, seed=41, device="cuda")
    st = W.make_signal_state(cfg, seed=41, device="cuda")
    announce(f"fused step parity {name} B={step.B} N={step.N}")
    h0, hd0, c0 = st.hist.cpu().numpy(), st.head.cpu().numpy(), st.count.cpu().numpy()
    f = gpu_lib.step(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                     step.u_acc, step.u_res, step.k_max, st.hist, st.head, st.count, st.sl_max)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in f.items()}
    host = W.host_arrays(step)
    smax = st.sl_max.cpu().numpy().astype(np.float64)
    ref, sr, nr, spread = oracle_chain(host, h0, hd0, c0, smax, step.k_max)
    rep = compare_verify(got, ref, host["sl"], host["cu_sl"], f"step {name}", host=host)
    compare_signal({**got, "seq_err": got["seq_err"].astype(np.uint32) & 96}, sr, f"step {name} signal", spread)
    rep["sl_ties"] = compare_sl(got, nr, sr, spread, smax, step.k_max, f"step {name}")
    print(f"[report] fused step {name}: {rep}", flush=True)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("shape", ["reduced", "full"])
def test_resume_from_snapshot(gpu_lib, shape):
    """Checkpoint and resume of the controller state: restarting a run of
    dsde_step from a copy of (hist, head, count) taken midway, in fresh
    buffers, reproduces the uninterrupted run bit for bit.  Full shape:
    B = 1024, V = 128256, 60 steps from empty rings with the snapshot at step
    40, after every ring (W = 32) has filled and wrapped."""
    if shape == "full":
        cfg, seed, steps, cut = W.CONFIGS["loop"], 9, 60, 40
    else:
        cfg, seed, steps, cut = dict(W.CONFIGS["loop"], B=128, V=4096), 8, 10, 4
    announce(f"resume B={cfg['B']} V={cfg['V']} {steps} steps, snapshot at {cut}")
    st = W.make_signal_state(cfg, seed=seed, device="cuda")
    sl, sigma = W.sample_sl(cfg, seed), W.initial_sigma(cfg, seed)

    def one(st_, t, sl_, sigma_):
        step = W.make_step(cfg, seed=seed, device="cuda", step=t, sl=sl_, sigma=sigma_)
        f = gpu_lib.step(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                         step.u_acc, step.u_res, step.k_max, st_.hist, st_.head, st_.count, st_.sl_max)
        torch.cuda.synchronize()
        return {k: v.clone() for k, v in f.items()}

    full, snap = {}, None
    for t in range(steps):
        if t == cut:
            snap = (clone_state(st), sl.copy(), sigma.copy())
            if shape == "full":
                assert (st.count.cpu().numpy() == cfg["W"]).all()
        f = one(st, t, sl, sigma)
        if t >= cut:
            full[t] = f
        if t % 10 == 0:
            print(f"[case] resume {shape}: uninterrupted step {t}", flush=True)
        sl, sigma = f["sl_next"].cpu().numpy(), W.walk_sigma(sigma, cfg, seed, t)
    st2, sl, sigma = snap
    for t in range(cut, steps):
        f = one(st2, t, sl, sigma)
        for k, v in f.items():
            a, b = v, full[t][k]
            if a.dtype.is_floating_point:
                a, b = a.view(torch.int32), b.view(torch.int32)
            assert torch.equal(a, b), f"step {t}: {k} differs after resume"
        sl, sigma = f["sl_next"].cpu().numpy(), W.walk_sigma(sigma, cfg, seed, t)
    assert torch.equal(st2.hist.view(torch.int32), st.hist.view(torch.int32))
    assert torch.equal(st2.head, st.head) and torch.equal(st2.count, st.count)


@pytest.mark.parametrize("name", ["b64", "greedy"])
def test_sl_max_calibration(gpu_lib, name):
    """Eq. 1 over four calibration steps, per sequence and pooled, against the
    oracle's Eq. 1 on the oracle's own verification of the same inputs
    (sequences with an acceptance or draw tie in any step are left out)."""
    cfg = W.CONFIGS[name]
    announce(f"SL_max calibration {name}")
    B = cfg["B"]
    state = gpu_lib.new_calibration_state(B)
    acc_ref = [[] for _ in range(B)]
    kld_ref = [[] for _ in range(B)]
    tie = np.zeros(B, bool)
    for t in range(4):
        step = W.make_step(cfg, seed=70 + t, device="cuda")
        v = gpu_lib.verify(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                           step.u_acc, step.u_res, step.k_max)
        gpu_lib.calibration_update(step.sl, step.cu_sl, v["accepted"], v["kld"], v["seq_err"], state)
        host = W.host_arrays(step)
        ref = oracle.verify(**host, n_threads=16)
        tie |= ref["acc_tie"] != 0  # a draw tie changes the emitted token, not the count
        cu = host["cu_sl"]
        for b in range(B):
            acc_ref[b].append(int(ref["accepted"][b]))
            kld_ref[b].extend(ref["kld"][cu[b]:cu[b + 1]].tolist())
    per = gpu_lib.calibrate_sl_max(state, eps=1e-6).cpu().numpy()
    pooled = gpu_lib.calibrate_sl_max(state, eps=1e-6, pooled=True).cpu().numpy()
    want = np.array([oracle.calibrate_sl_max(acc_ref[b], kld_ref[b]) for b in range(B)])
    ok = ~tie
    np.testing.assert_allclose(per[ok], want[ok], rtol=1e-4)
    # pooled: the KLD part does not depend on the acceptance decisions, and the
    # pooled SL_A,max is fixed whenever no tie can move the batch maximum
    allk = [k for b in range(B) for k in kld_ref[b]]
    a_free = max(max(acc_ref[b]) for b in range(B) if ok[b])
    a_all = max(max(a) for a in acc_ref)
    if not tie.any() or a_free == cfg["k_max"]:
        want_pooled = oracle.calibrate_sl_max([a_all if not tie.any() else a_free], allk)
        np.testing.assert_allclose(pooled, want_pooled, rtol=1e-4)
    else:
        print(f"[report] calibration {name}: pooled value left unchecked (tie at the maximum)", flush=True)
    assert np.all(pooled == pooled[0])
    print(f"[report] calibration {name}: compared {int(ok.sum())} of {B}, pooled SL_max {pooled[0]:.4f}",
          flush=True)
