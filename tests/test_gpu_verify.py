"""GPU parity of dsde_verify against the CPU oracle (through the C ABI).

Inputs are seeded and synthetic (workloads.py); the oracle receives a host copy
of the very same device inputs.  Every case prints its name before it runs.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from tests.helpers import bf16_bits, packed_layout
from tests.parity import compare_verify, run_verify

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"\n[case] {msg}", flush=True)


def check_step(dsde, step, label, n_threads=16):
    announce(f"{label}: B={step.B} N={step.N} V={step.V} dtype={step.target.dtype}")
    got = run_verify(dsde, step)
    ref = oracle.verify(**W.host_arrays(step), n_threads=n_threads)
    host = W.host_arrays(step)
    rep = compare_verify(got, ref, host["sl"], host["cu_sl"], label, host=host)
    print(f"[report] {label}: {rep}", flush=True)
    return got, ref, rep


def step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, k_max, dtype="bf16", device="cuda"):
    sl, cu = packed_layout(sls)
    tt = torch.float32 if dtype == "fp32" else torch.bfloat16

    def dev(x):
        return torch.as_tensor(np.ascontiguousarray(x), device=device)
    return W.Step(target=dev(target.astype(np.float32)).to(tt), draft=dev(draft.astype(np.float32)).to(tt),
                  sl=dev(sl), cu_sl=dev(cu), draft_tokens=dev(np.asarray(tokens, np.int32)),
                  temperature=dev(np.asarray(temps, np.float32)), u_acc=dev(np.asarray(u_acc, np.float32)),
                  u_res=dev(np.asarray(u_res, np.float32)), k_max=k_max)


def random_arrays(rng, sls, V, sigma=2.0, noise=1.0):
    sl, cu = packed_layout(sls)
    B, N = len(sls), int(cu[-1])
    target = rng.normal(0, sigma, (N + B, V)).astype(np.float32)
    seq = np.repeat(np.arange(B), sls)
    draft = (target[np.arange(N) + seq] + rng.normal(0, noise, (N, V))).astype(np.float32)
    tokens = rng.integers(0, V, N)
    return target, draft, tokens, rng.random(N).astype(np.float32), rng.random(B).astype(np.float32)


@pytest.mark.parametrize("name", ["tiny", "b64", "b256", "lowacc", "greedy", "b256g"])
def test_workload_parity(gpu_lib, name):
    cfg = W.CONFIGS[name]
    step = W.make_step(cfg, seed=11, device="cuda")
    _, ref, rep = check_step(gpu_lib, step, f"workload {name}")
    assert rep["compared"] >= 0.9 * step.B


@pytest.mark.parametrize("V", [1, 2, 17, 100, 8191, 8200, 16392, 32001])
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_vocab_edges(gpu_lib, V, dtype):
    rng = np.random.default_rng(V)
    sls = [3, 0, 1, 5, 2, 0, 4]
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V, noise=0.7)
    step = step_from_arrays(target, draft, sls, tokens, [1.0, 0.7, 1.3, 1.0, 0.5, 2.0, 1.0], u_acc, u_res, 5,
                            dtype)
    check_step(gpu_lib, step, f"vocab V={V} {dtype}")


@pytest.mark.parametrize("V,dtype", [(600000, "bf16"), (600001, "bf16"), (600000, "fp32"), (4194304, "bf16")])
def test_large_vocab(gpu_lib, V, dtype):
    """More than 64 chunks per row (two rounds of the chunk walk, several chunks
    per combining lane) up to the largest supported vocabulary."""
    rng = np.random.default_rng(V % 1000 + 17)
    sls = [3, 0, 2, 1] if V < 4194304 else [1, 1]
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V, noise=0.3)
    temps = [1.0, 0.8, 1.1, 0.6][:len(sls)]
    step = step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, 3, dtype)
    check_step(gpu_lib, step, f"large vocab V={V} {dtype}")


@pytest.mark.parametrize("V,dtype", [(300, "bf16"), (512, "bf16"), (512, "fp32"), (301, "fp32")])
def test_large_batch(gpu_lib, V, dtype):
    """More sequences than CUs and than the set-up kernel has threads (the
    256-thread per-sequence kernel and the set-up's looping path), ragged SL
    including 0, mixed temperatures and greedy sequences; vectorised (V a
    multiple of the vector width) and scalar row paths."""
    rng = np.random.default_rng(1500 + V)
    B = 1500
    sls = rng.integers(0, 4, B).tolist()
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V, noise=0.8)
    temps = rng.choice([0.0, 0.7, 1.0, 1.3], B).tolist()
    step = step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, 3, dtype)
    _, _, rep = check_step(gpu_lib, step, f"large batch B={B} V={V} {dtype}")
    assert rep["compared"] >= 0.9 * B


def test_nothing_drafted(gpu_lib):
    rng = np.random.default_rng(3)
    V = 5000
    target = rng.normal(0, 2, (6, V)).astype(np.float32)
    step = step_from_arrays(target, np.zeros((0, V), np.float32), [0] * 6, [], [1.0] * 6, [], rng.random(6), 4)
    got, _, rep = check_step(gpu_lib, step, "all SL = 0")
    assert (got["accepted"] == 0).all() and rep["compared"] + rep["cdf_ties"] == 6


def test_identical_rows_accept_everything_with_zero_kld(gpu_lib):
    rng = np.random.default_rng(4)
    sls = [4, 2, 3]
    V = 12345
    target, _, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    sl, cu = packed_layout(sls)
    seq = np.repeat(np.arange(3), sls)
    draft = target[np.arange(cu[-1]) + seq]
    u_acc = np.full(cu[-1], np.float32(np.nextafter(np.float32(1), np.float32(0))))
    step = step_from_arrays(target, draft, sls, tokens, [1.0, 0.8, 1.2], u_acc, u_res, 4)
    got, _, _ = check_step(gpu_lib, step, "identical rows")
    assert (got["accepted"] == np.array(sls)).all()
    assert (got["kld"] == 0.0).all()


def test_peaked_distributions(gpu_lib):
    rng = np.random.default_rng(5)
    sls = [3, 3, 3, 3]
    V = 20000
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    target[:, 77] += 60.0            # p is one-hot at 77
    draft[0::2, 77] += 60.0          # q one-hot at 77 on even positions
    draft[1::2, 123] += 60.0         # and at 123 on odd ones
    tokens[:] = np.where(np.arange(len(tokens)) % 2 == 0, 77, 123)
    step = step_from_arrays(target, draft, sls, tokens, [1.0] * 4, u_acc, u_res, 3)
    check_step(gpu_lib, step, "peaked p and q")


def test_error_contract(gpu_lib):
    rng = np.random.default_rng(6)
    sls = [2, 2, 2, 2, 2, 2, 2]
    V = 9000
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    temps = np.ones(7, np.float32)
    tokens[2] = V                  # seq 1: token out of range
    u_acc[4] = 1.0                 # seq 2: uniform out of [0, 1)
    temps[3] = 2.0 ** 17           # seq 3: temperature outside [2^-16, 2^16]
    draft[8, 17] = np.nan          # seq 4: NaN in a drafted pair
    target[5 * 3 + 1, 40] = -np.inf  # seq 5: -inf in a drafted target row
    # seq 6: both drafts accepted (equal rows, u just below 1), bonus row has +inf
    target[6 * 3: 6 * 3 + 2] = draft[12:14]
    u_acc[12:14] = 0.99999
    target[6 * 3 + 2, 5] = np.inf
    step = step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, 2)
    got, ref, _ = check_step(gpu_lib, step, "error contract")
    assert list(got["seq_err"]) == [0, 2, 16, 8, 4, 4, 4]
    assert np.isnan(got["kld"][2:12]).all() and np.isfinite(got["kld"][:2]).all()
    assert np.isfinite(got["kld"][12:14]).all()  # a bad bonus row withholds only the token


def test_bad_layout(gpu_lib):
    rng = np.random.default_rng(7)
    sls = [2, 3, 1]
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, 500)
    step = step_from_arrays(target, draft, sls, tokens, [1.0] * 3, u_acc, u_res, 3)
    cu = step.cu_sl.clone()
    cu[1] += 1
    step.cu_sl = cu
    announce("bad layout")
    got = run_verify(gpu_lib, step, row_lse=False)
    assert (got["seq_err"] == 1).all() and (got["accepted"] == 0).all() and (got["tokens"] == -1).all()


def test_unaligned_rows_take_the_scalar_path(gpu_lib):
    rng = np.random.default_rng(8)
    sls = [3, 1, 4]
    V = 4096
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V, noise=0.5)
    step = step_from_arrays(target, draft, sls, tokens, [1.0, 0.7, 1.0], u_acc, u_res, 4)
    # the same logits, one element past a 16-byte boundary
    tb = torch.empty(step.target.numel() + 1, dtype=torch.bfloat16, device="cuda")
    db = torch.empty(step.draft.numel() + 1, dtype=torch.bfloat16, device="cuda")
    tb[1:].copy_(step.target.reshape(-1))
    db[1:].copy_(step.draft.reshape(-1))
    shifted = W.Step(**{**step.__dict__, "target": tb[1:].view(step.target.shape),
                        "draft": db[1:].view(step.draft.shape)})
    check_step(gpu_lib, shifted, "unaligned rows")


@pytest.mark.parametrize("name", ["tiny", "b64", "b256", "lowacc", "greedy", "b256g"])
def test_deterministic(gpu_lib, name):
    """Run-to-run bitwise reproducibility of dsde_verify (every reduction has a
    fixed order)."""
    step = W.make_step(W.CONFIGS[name], seed=12, device="cuda")
    announce(f"determinism {name} B={step.B} N={step.N}")
    a = run_verify(gpu_lib, step)
    b = run_verify(gpu_lib, step)
    for k in ("accepted", "tokens", "seq_err", "row_lse"):
        assert np.array_equal(a[k], b[k]), k
    for k in ("kld", "draft_entropy"):
        assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), k


@pytest.mark.parametrize("name", ["b64", "lowacc", "b256g"])
def test_entropy_request_changes_nothing_else(gpu_lib, name):
    """A call that asks for no draft entropy runs the statistics kernel without
    the entropy accumulator; every other output is the same bit for bit as in
    a call that asks for it."""
    import torch
    step = W.make_step(W.CONFIGS[name], seed=14, device="cuda")
    announce(f"entropy request {name} B={step.B} N={step.N}")
    runs = []
    for ent in (True, False):
        lse = torch.empty((max(step.N, 1), 2), dtype=torch.float64, device="cuda")[:step.N]
        out = gpu_lib.verify(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                             step.u_acc, step.u_res, step.k_max, row_lse=lse, draft_entropy=ent)
        torch.cuda.synchronize()
        res = {k: v.cpu().numpy() for k, v in out.items()}
        res["row_lse"] = lse.cpu().numpy()
        runs.append(res)
    a, b = runs
    assert "draft_entropy" in a and "draft_entropy" not in b
    for k in ("accepted", "tokens", "seq_err", "row_lse"):
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(a["kld"].view(np.uint32), b["kld"].view(np.uint32))


@pytest.mark.parametrize("name", ["b64", "b256", "lowacc", "b256g"])
def test_fused_step_deterministic(gpu_lib, name):
    """dsde_step twice from the same controller state: every output and the
    updated ring identical bit for bit."""
    import torch
    cfg = W.CONFIGS[name]
    step = W.make_step(cfg, seed=13, device="cuda")
    st = W.make_signal_state(cfg, seed=13, device="cuda")
    announce(f"fused step determinism {name} B={step.B} N={step.N}")
    runs = []
    for _ in range(2):
        s = W.SignalState(hist=st.hist.clone(), head=st.head.clone(), count=st.count.clone(), sl_max=st.sl_max)
        f = gpu_lib.step(step.target, step.draft, step.sl, step.cu_sl, step.draft_tokens, step.temperature,
                         step.u_acc, step.u_res, step.k_max, s.hist, s.head, s.count, s.sl_max, draft_entropy=True)
        torch.cuda.synchronize()
        runs.append(({k: v.clone() for k, v in f.items()}, s))
    (a, sa), (b, sb) = runs
    for k in a:
        x, y = a[k], b[k]
        if x.dtype.is_floating_point:
            x, y = x.view(torch.int32), y.view(torch.int32)
        assert torch.equal(x, y), k
    assert torch.equal(sa.hist.view(torch.int32), sb.hist.view(torch.int32))
    assert torch.equal(sa.head, sb.head) and torch.equal(sa.count, sb.count)


def test_draw_distribution_matches_target(gpu_lib):
    """Speculative-sampling theorem on the GPU: over a grid of uniforms the
    emitted first token is distributed as p (no oracle involved)."""
    V, M = 7, 64
    zt = np.array([0.5, -1.0, 1.5, 0.0, -0.3, 0.9, -2.0], np.float32)
    zd = np.array([-0.4, 0.8, 0.3, 1.1, -1.5, 0.2, 0.6], np.float32)
    p = np.exp(zt.astype(np.float64)); p /= p.sum()
    q = np.exp(zd.astype(np.float64)); q /= q.sum()
    g = ((np.arange(M) + 0.5) / M).astype(np.float32)
    xs, us, ur, wt = [], [], [], []
    for x in range(V):
        for u in g:
            for u2 in g:
                xs.append(x), us.append(u), ur.append(u2), wt.append(q[x] / (M * M))
    B = len(xs)
    target = np.empty((2 * B, V), np.float32)
    target[0::2] = zt
    target[1::2] = zt
    step = step_from_arrays(target, np.tile(zd, (B, 1)), [1] * B, xs, [1.0] * B, us, ur, 1, "fp32")
    announce(f"draw distribution B={B}")
    got = run_verify(gpu_lib, step, row_lse=False)
    dist = np.zeros(V)
    np.add.at(dist, got["tokens"][:, 0], np.asarray(wt))
    np.testing.assert_allclose(dist, p, atol=2.0 / M)


def test_constructed_ties(gpu_lib):
    """Acceptance uniforms set to p(x)/q(x) itself (nearest fp32), and draw
    uniforms that put u' * Z exactly on a CDF boundary of uniform logits: the
    oracle flags these as ties; the GPU must emit a valid draw for each, and
    match the oracle exactly on the interleaved sequences without a tie."""
    rng = np.random.default_rng(9)
    V, B = 50, 96
    sls = [1] * 64 + [0] * 32
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V, noise=0.8)
    sl, cu = packed_layout(sls)
    for b in range(0, 64, 2):  # even sequences: u on the acceptance boundary
        j = cu[b]
        p = np.exp(target[j + b].astype(np.float64))
        p /= p.sum()
        q = np.exp(draft[j].astype(np.float64))
        q /= q.sum()
        r = p[tokens[j]] / q[tokens[j]]
        u_acc[j] = np.float32(min(r, 1.0 - 2.0 ** -24))
    # bonus draws over uniform logits: C(k) = k/4 exactly for V = 4 tokens
    tgt = np.vstack([target[:cu[64] + 64], np.zeros((32, V), np.float32)])
    tgt[cu[64] + 64:, 4:] = -60.0  # only the first four tokens carry mass
    u_res[64:] = np.tile(np.array([0.25, 0.5, 0.75, 0.3], np.float32), 8)
    step = step_from_arrays(tgt, draft, sls, tokens, [1.0] * B, u_acc, u_res, 1, "fp32")
    _, ref, rep = check_step(gpu_lib, step, "constructed ties")
    assert rep["acc_ties"] >= 24 and rep["cdf_ties"] >= 24, rep


@pytest.mark.parametrize("V,dtype", [(3 * 8192 + 704, "bf16"), (3 * 8192 + 704, "fp32"), (3 * 8192 + 705, "bf16"),
                                     (3 * 8192 + 705, "fp32")])
def test_draw_at_sub_block_and_chunk_boundaries(gpu_lib, V, dtype):
    """The draw's three levels (chunk of 8192, sub-block of 512, element) at
    their edges: all mass on tokens that open or close a sub-block or a chunk,
    up to the last token of a partial last chunk, and u' in the middle of each
    token's CDF interval.  Every sequence rejects its one draft (q is one-hot on
    a token p does not hold) or accepts it and draws from the bonus row, so the
    residual and the bonus draws are both checked, against the oracle and
    against the token the construction fixes.  V = 8k + 704 takes the
    vectorised paths, V = 8k + 705 the scalar ones."""
    hot = np.array([0, 511, 512, 1023, 4095, 8191, 8192, 8703, 16383, 16384, 24575, 24576, V - 1])
    H = len(hot)
    B = 2 * H
    sls = [1] * B
    rng = np.random.default_rng(V)
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    other = 3000  # not a hot token
    for b in range(B):
        i = b % H
        row = np.full(V, -30.0, np.float32)
        row[hot] = 0.0
        if b < H:  # reject: q one-hot on `other`, p spread evenly over the hot tokens
            target[2 * b] = row
            draft[b] = -30.0
            draft[b, other] = 30.0
            tokens[b] = other
            u_acc[b] = 0.5
        else:      # accept (equal rows), then the bonus row holds the hot tokens
            draft[b] = target[2 * b]
            tokens[b] = other
            u_acc[b] = 0.0
            target[2 * b + 1] = row
        u_res[b] = (i + 0.5) / H
    step = step_from_arrays(target, draft, sls, tokens, [1.0] * B, u_acc, u_res, 1, dtype)
    got, ref, rep = check_step(gpu_lib, step, f"draw at boundaries V={V} {dtype}")
    assert rep["compared"] == B, rep
    want = np.concatenate([hot, hot])
    assert (got["accepted"] == np.array([0] * H + [1] * H)).all()
    drawn = got["tokens"][np.arange(B), got["accepted"]]
    assert (drawn == want).all(), (drawn, want)


@pytest.mark.parametrize("V,dtype", [(5000, "bf16"), (5000, "fp32"), (8200, "bf16"), (600000, "bf16")])
def test_greedy_ties_and_emissions(gpu_lib, V, dtype):
    """Greedy verification (T = 0) with repeated maxima inside and across
    chunks: the argmax is the smallest token id holding the maximum; drafts hit
    it, miss it, or sit on a later tied maximum."""
    rng = np.random.default_rng(V % 997 + 3)
    sls = [3, 2, 4, 0, 1, 5]
    sl, cu = packed_layout(sls)
    B = len(sls)
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V, noise=0.8)
    for r in range(target.shape[0]):
        m = np.float32(target[r].max() + 2.0)
        cols = np.sort(rng.choice(V, 3, replace=False))  # three equal maxima, maybe in different chunks
        target[r, cols] = m
    for b, s in enumerate(sls):
        for j in range(s):
            r = cu[b] + b + j
            ties = np.nonzero(target[r] == target[r].max())[0]
            pick = rng.integers(0, 3)
            tokens[cu[b] + j] = ties[0] if pick == 0 else (ties[-1] if pick == 1 else (ties[0] + 1) % V)
    temps = np.zeros(B, np.float32)
    temps[1::3] = 1.0  # a few sampling sequences in between
    step = step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, 5, dtype)
    got, ref, rep = check_step(gpu_lib, step, f"greedy ties V={V} {dtype}")
    assert rep["compared"] + rep["acc_ties"] + rep["cdf_ties"] >= B - 1


def test_greedy_ignores_uniforms_and_flags_a_bad_bonus_row(gpu_lib):
    rng = np.random.default_rng(51)
    sls = [2, 2, 3]
    V = 3000
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    sl, cu = packed_layout(sls)
    for b, s in enumerate(sls):  # every draft is the target argmax: all accepted, bonus sampled
        for j in range(s):
            tokens[cu[b] + j] = int(np.argmax(target[cu[b] + b + j]))
    u_acc[:] = 7.0   # not in [0, 1): unused by greedy sequences
    u_res[:] = -1.0
    target[cu[2] + 2 + 3, 11] = np.inf  # sequence 2's bonus row
    step = step_from_arrays(target, draft, sls, tokens, [0.0, 0.0, 0.0], u_acc, u_res, 3)
    got, ref, _ = check_step(gpu_lib, step, "greedy: unused uniforms, bad bonus row")
    assert list(got["seq_err"]) == [0, 0, 4]
    assert list(got["accepted"][:2]) == [2, 2]
    assert np.isfinite(got["kld"]).all()


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_longest_speculation(gpu_lib, dtype):
    """k_max = DSDE_MAX_K = 63: a sequence drafting 63 tokens that all pass
    (identical rows, bonus draw from row 63), one with a long accepted run
    ending in a rejection, a greedy one rejecting at position 40, and SL = 0
    and a short sequence beside them; unsharded and over three slices."""
    rng = np.random.default_rng(63)
    V, k_max = 9000, 63
    sls = [63, 0, 17, 63, 63]
    target, draft, tokens, u_acc, u_res = random_arrays(rng, sls, V)
    sl, cu = packed_layout(sls)
    draft[cu[0]:cu[1]] = target[0:63]                                  # seq 0: p = q
    u_acc[cu[0]:cu[1]] = 0.999
    draft[cu[3]:cu[4]] = target[cu[3] + 3:cu[4] + 3] + rng.normal(0, 0.02, (63, V))  # seq 3: q close to p
    u_acc[cu[3]:cu[4]] = 0.05
    u_acc[cu[3] + 50] = 0.99999                                          # a likely rejection late in the run
    temps = [1.0, 0.7, 0.9, 1.0, 0.0]
    step = step_from_arrays(target, draft, sls, tokens, temps, u_acc, u_res, k_max, dtype)
    # seq 4 (greedy): draft the target argmax of rows 0..39, then a token that is not
    rows = step.target[cu[4] + 4:cu[4] + 4 + 63].float().cpu().numpy()
    greedy_tok = rows.argmax(axis=1).astype(np.int32)
    greedy_tok[40] = (greedy_tok[40] + 1) % V
    toks = step.draft_tokens.clone()
    toks[cu[4]:cu[5]] = torch.as_tensor(greedy_tok, device="cuda")
    step = W.Step(**{**step.__dict__, "draft_tokens": toks})
    got, _, rep = check_step(gpu_lib, step, f"k_max 63 {dtype}")
    assert got["accepted"][0] == 63 and got["accepted"][4] == 40, got["accepted"]
    assert got["accepted"][3] > 10, got["accepted"]
    assert rep["errored"] == 0
    import paper_2509_01083_amd as dsde
    from tests.test_gpu_shard import check_sharded
    check_sharded(dsde, step, dsde.slice_bounds(V, 3), f"k_max 63 {dtype} sharded")
