"""Pins of the CPU oracle against facts fixed by mathematics and the paper.

Each check is independent of the oracle's own code: closed forms, library
routines (scipy/numpy) on special cases, invariants, and brute force on tiny
vocabularies.  A plausible slip in the oracle (a dropped temperature, the KL
direction reversed, a wrong row index, a sign error in the residual, an
off-by-one in the window) fails at least one of them.
"""
import math

import numpy as np
import pytest
from scipy.optimize import minimize_scalar
from scipy.special import logsumexp, softmax
from scipy.stats import entropy

from tests.helpers import bf16_bits, packed_layout, single_pair_batch

U_MAX = np.float32(np.nextafter(np.float32(1.0), np.float32(0.0)))  # largest fp32 below 1


def run_single(orc, zt, zd, x=0, u=0.5, u_res=0.5, T=1.0, bonus=None):
    kw = single_pair_batch(zt, zd, [x], [u], [u_res], temperature=T, bonus_logits=bonus)
    return orc.verify(**kw)


# ---------------------------------------------------------------- softmax / lse

def test_lse_matches_logsumexp_with_temperature(orc):
    rng = np.random.default_rng(1)
    for T in (1.0, 0.7, 1.9):
        zt = rng.normal(0, 3, 97).astype(np.float32)
        zd = rng.normal(0, 3, 97).astype(np.float32)
        out = run_single(orc, zt, zd, T=T)
        Tf = float(np.float32(T))
        assert out["lse"][0, 0] == pytest.approx(logsumexp(zt.astype(np.float64) / Tf), abs=1e-12)
        assert out["lse"][0, 1] == pytest.approx(logsumexp(zd.astype(np.float64) / Tf), abs=1e-12)


def test_lse_special_cases(orc):
    # V = 1: lse = z, p = 1
    out = run_single(orc, [2.5], [-1.0])
    assert out["lse"][0, 0] == 2.5 and out["lse"][0, 1] == -1.0
    assert out["kld"][0] == 0.0
    # uniform logits: lse = c + ln V
    out = run_single(orc, np.full(40, 3.0), np.full(40, -2.0))
    assert out["lse"][0, 0] == pytest.approx(3.0 + math.log(40), abs=1e-13)
    assert out["lse"][0, 1] == pytest.approx(-2.0 + math.log(40), abs=1e-13)


# ---------------------------------------------------------------- KL divergence

def test_kl_zero_for_identical_and_shifted_logits(orc):
    rng = np.random.default_rng(2)
    z = rng.normal(0, 4, 300).astype(np.float32)
    assert run_single(orc, z, z)["kld"][0] == 0.0
    out = run_single(orc, z, z - np.float32(8.0))  # softmax is shift invariant
    assert abs(out["kld"][0]) < 1e-12


def test_kl_two_token_closed_form_and_direction(orc):
    zt = np.array([0.3, -1.2], np.float32)
    zd = np.array([-0.8, 0.9], np.float32)
    p0 = 1.0 / (1.0 + math.exp(float(zt[1]) - float(zt[0])))
    q0 = 1.0 / (1.0 + math.exp(float(zd[1]) - float(zd[0])))
    kl_pq = p0 * math.log(p0 / q0) + (1 - p0) * math.log((1 - p0) / (1 - q0))
    kl_qp = q0 * math.log(q0 / p0) + (1 - q0) * math.log((1 - q0) / (1 - p0))
    got = run_single(orc, zt, zd)["kld"][0]
    assert got == pytest.approx(kl_pq, rel=1e-12)
    assert abs(got - kl_qp) > 1e-3  # the direction is KL(target || draft)


@pytest.mark.parametrize("T", [1.0, 0.7])
def test_kl_matches_scipy_entropy(orc, T):
    rng = np.random.default_rng(3)
    zt = rng.normal(0, 3, 500).astype(np.float32)
    zd = (zt + rng.normal(0, 1, 500)).astype(np.float32)
    Tf = float(np.float32(T))
    p = softmax(zt.astype(np.float64) / Tf)
    q = softmax(zd.astype(np.float64) / Tf)
    assert run_single(orc, zt, zd, T=T)["kld"][0] == pytest.approx(entropy(p, q), rel=1e-10)


def test_kl_gaussian_in_logit_closed_form(orc):
    # z_v = -(v - mu)^2 / (2 sigma^2) on a lattice wide enough that the discrete
    # Gaussians equal the continuous ones to far below the tolerance
    V = 256
    v = np.arange(V, dtype=np.float64)
    m1, s1, m2, s2 = 128.0, 1.5, 128.7, 2.0
    zt = (-(v - m1) ** 2 / (2 * s1 ** 2)).astype(np.float32)
    zd = (-(v - m2) ** 2 / (2 * s2 ** 2)).astype(np.float32)
    kl = math.log(s2 / s1) + (s1 ** 2 + (m1 - m2) ** 2) / (2 * s2 ** 2) - 0.5
    assert run_single(orc, zt, zd)["kld"][0] == pytest.approx(kl, abs=2e-6)


def test_kl_nonnegative_and_pinsker(orc):
    rng = np.random.default_rng(4)
    for _ in range(20):
        zt = rng.normal(0, 2, 64).astype(np.float32)
        zd = rng.normal(0, 2, 64).astype(np.float32)
        kl = run_single(orc, zt, zd)["kld"][0]
        tv = 0.5 * np.abs(softmax(zt.astype(np.float64)) - softmax(zd.astype(np.float64))).sum()
        assert kl >= 0.0
        assert tv <= math.sqrt(kl / 2) + 1e-12


# ---------------------------------------------------------------- acceptance and draw

def _grid(M):
    return ((np.arange(M) + 0.5) / M).astype(np.float32)


def test_acceptance_probability_is_one_minus_tv(orc):
    rng = np.random.default_rng(5)
    V, M = 8, 2000
    zt = rng.normal(0, 1.5, V).astype(np.float32)
    zd = rng.normal(0, 1.5, V).astype(np.float32)
    p = softmax(zt.astype(np.float64))
    q = softmax(zd.astype(np.float64))
    xs = np.repeat(np.arange(V), M)
    us = np.tile(_grid(M), V)
    out = orc.verify(**single_pair_batch(zt, zd, xs, us, np.full(V * M, 0.5)))
    acc = out["accepted"].reshape(V, M).mean(axis=1)
    np.testing.assert_allclose(acc, np.minimum(1.0, p / q), atol=1.0 / M + 1e-12)
    assert float(q @ acc) == pytest.approx(1.0 - 0.5 * np.abs(p - q).sum(), abs=1.0 / M)


def test_draw_is_normalised_residual_and_output_is_target(orc):
    rng = np.random.default_rng(6)
    V, M, Mr = 6, 1000, 4000
    zt = rng.normal(0, 1.5, V).astype(np.float32)
    zd = rng.normal(0, 1.5, V).astype(np.float32)
    p = softmax(zt.astype(np.float64))
    q = softmax(zd.astype(np.float64))
    # acceptance per drafted token
    out = orc.verify(**single_pair_batch(zt, zd, np.repeat(np.arange(V), M), np.tile(_grid(M), V),
                                         np.full(V * M, 0.5)))
    acc = out["accepted"].reshape(V, M).mean(axis=1)
    # residual draw: a token that is always rejected at u just below 1
    x_rej = int(np.argmin(p / q))
    out = orc.verify(**single_pair_batch(zt, zd, [x_rej] * Mr, [U_MAX] * Mr, _grid(Mr)))
    assert (out["accepted"] == 0).all()
    resid = np.maximum(p - q, 0.0)
    assert out["sample_mass"][0] == pytest.approx(resid.sum(), rel=1e-12)  # Z = TV
    R = np.bincount(out["tokens"][:, 0], minlength=V) / Mr
    np.testing.assert_allclose(R, resid / resid.sum(), atol=V / Mr)
    # speculative-sampling theorem: the emitted token is distributed as p
    emitted = q * acc + (q @ (1.0 - acc)) * R
    np.testing.assert_allclose(emitted, p, atol=2.0 / M + 2.0 * V / Mr)


def test_brute_force_emitted_distribution_tiny_vocab(orc):
    V, M = 3, 100
    zt = np.array([0.4, -0.7, 1.1], np.float32)
    zd = np.array([1.3, -0.2, -0.5], np.float32)
    p = softmax(zt.astype(np.float64))
    q = softmax(zd.astype(np.float64))
    xs, us, ur, wt = [], [], [], []
    g = _grid(M)
    for x in range(V):
        for u in g:
            for u2 in g:
                xs.append(x), us.append(u), ur.append(u2), wt.append(q[x] / (M * M))
    out = orc.verify(**single_pair_batch(zt, zd, xs, us, ur))
    dist = np.zeros(V)
    np.add.at(dist, out["tokens"][:, 0], np.asarray(wt))
    np.testing.assert_allclose(dist, p, atol=2.0 / M)


def test_bonus_draw_follows_bonus_row(orc):
    V, Mr = 5, 4000
    zt = np.array([0.0, 1.0, -1.0, 0.5, 2.0], np.float32)
    bonus = np.array([1.5, -0.5, 0.3, 0.0, -2.0], np.float32)
    out = orc.verify(**single_pair_batch(zt, zt, [4] * Mr, [0.0] * Mr, _grid(Mr), bonus_logits=bonus))
    assert (out["accepted"] == 1).all()
    assert (out["tokens"][:, 0] == 4).all()
    D = np.bincount(out["tokens"][:, 1], minlength=V) / Mr
    np.testing.assert_allclose(D, softmax(bonus.astype(np.float64)), atol=V / Mr)


def test_equal_distributions_always_accept_and_zero_target_mass_rejects(orc):
    z = np.array([0.2, -0.3, 0.9, 0.0], np.float32)
    out = orc.verify(**single_pair_batch(z, z, [0, 1, 2, 3], [U_MAX] * 4, [0.5] * 4))
    assert (out["accepted"] == 1).all()
    zt = np.array([0.0, -2000.0, 0.0, 0.0], np.float32)  # p(1) underflows to 0
    out = orc.verify(**single_pair_batch(zt, z, [1] * 3, [0.0, 0.5, 0.9], [0.5] * 3))
    assert (out["accepted"] == 0).all()
    assert (out["tokens"][:, 0] != 1).all()


def test_inverse_cdf_edges(orc):
    # bonus row uniform over 4 tokens: C(k) = (k + 1) / 4, exactly representable
    z = np.zeros(4, np.float32)
    out = orc.verify(**single_pair_batch(z, z, [0] * 5, [0.0] * 5, [0.0, 0.25, 0.5, 0.7, U_MAX]))
    np.testing.assert_array_equal(out["tokens"][:, 1], [0, 1, 2, 2, 3])
    np.testing.assert_array_equal(out["cdf_tie"], [1, 1, 1, 0, 1])
    # u' = 0 picks the first token with positive residual weight
    zt = np.array([-5.0, -5.0, 3.0, 0.0], np.float32)
    zd = np.array([2.0, 2.0, -1.0, 2.5], np.float32)
    out = orc.verify(**single_pair_batch(zt, zd, [0], [U_MAX], [0.0]))
    assert out["accepted"][0] == 0 and out["tokens"][0, 0] == 2


# ---------------------------------------------------------------- ragged layout

def _random_batch(rng, sls, V, T=1.0):
    sl, cu = packed_layout(sls)
    B, N = len(sls), int(cu[-1])
    target = rng.normal(0, 2, (N + B, V)).astype(np.float32)
    draft = rng.normal(0, 2, (N, V)).astype(np.float32)
    return dict(target=target, draft=draft, V=V, sl=sl, cu_sl=cu,
                draft_tokens=rng.integers(0, V, N).astype(np.int32),
                temperature=np.full(B, T, np.float32),
                u_acc=rng.random(N).astype(np.float32) * 0.6,
                u_res=rng.random(B).astype(np.float32), k_max=max(sls))


def test_batch_equals_sequences_run_alone(orc):
    rng = np.random.default_rng(7)
    sls = [0, 2, 3, 1, 4]
    kw = _random_batch(rng, sls, 50)
    out = orc.verify(**kw)
    cu = kw["cu_sl"]
    for b, s in enumerate(sls):
        one = dict(target=kw["target"][cu[b] + b: cu[b + 1] + b + 1], draft=kw["draft"][cu[b]: cu[b + 1]],
                   V=50, sl=[s], cu_sl=[0, s], draft_tokens=kw["draft_tokens"][cu[b]: cu[b + 1]],
                   temperature=kw["temperature"][b: b + 1], u_acc=kw["u_acc"][cu[b]: cu[b + 1]],
                   u_res=kw["u_res"][b: b + 1], k_max=max(sls))
        o1 = orc.verify(**one)
        assert o1["accepted"][0] == out["accepted"][b]
        np.testing.assert_array_equal(o1["tokens"][0], out["tokens"][b])
        np.testing.assert_array_equal(o1["kld"], out["kld"][cu[b]: cu[b + 1]])


def test_draw_uses_the_first_rejected_pair(orc):
    V, Mr = 6, 3000
    rng = np.random.default_rng(8)
    rows = rng.normal(0, 1.5, (4, V)).astype(np.float32)   # target rows 0..2 + bonus
    drafts = rng.normal(0, 1.5, (3, V)).astype(np.float32)
    p1, q1 = softmax(rows[1].astype(np.float64)), softmax(drafts[1].astype(np.float64))
    x1 = int(np.argmin(p1 / q1))
    target = np.tile(rows, (Mr, 1))
    draft = np.tile(drafts, (Mr, 1))
    sl, cu = packed_layout([3] * Mr)
    toks = np.tile(np.array([0, x1, 0], np.int32), Mr)
    u_acc = np.tile(np.array([0.0, U_MAX, 0.0], np.float32), Mr)
    out = orc.verify(target=target, draft=draft, V=V, sl=sl, cu_sl=cu, draft_tokens=toks,
                     temperature=np.ones(Mr, np.float32), u_acc=u_acc, u_res=_grid(Mr), k_max=3)
    assert (out["accepted"] == 1).all()
    assert (out["tokens"][:, 0] == 0).all() and (out["tokens"][:, 2:] == -1).all()
    resid = np.maximum(p1 - q1, 0.0)
    D = np.bincount(out["tokens"][:, 1], minlength=V) / Mr
    np.testing.assert_allclose(D, resid / resid.sum(), atol=V / Mr)


def test_bf16_input_equals_fp32_of_same_values(orc):
    rng = np.random.default_rng(9)
    kw = _random_batch(rng, [2, 3], 33)
    bits_t, bits_d = bf16_bits(kw["target"]), bf16_bits(kw["draft"])
    f_t = (bits_t.astype(np.uint32) << 16).view(np.float32)
    f_d = (bits_d.astype(np.uint32) << 16).view(np.float32)
    o16 = orc.verify(**{**kw, "target": bits_t, "draft": bits_d})
    o32 = orc.verify(**{**kw, "target": f_t, "draft": f_d})
    for k in ("accepted", "tokens", "kld"):
        np.testing.assert_array_equal(o16[k], o32[k])


# ---------------------------------------------------------------- error contract

def test_error_bits_and_fallback_outputs(orc):
    rng = np.random.default_rng(10)
    base = _random_batch(rng, [2, 2, 2, 2, 2, 2], 16)
    kw = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in base.items()}
    kw["draft_tokens"][2] = 16           # seq 1: token out of range
    kw["u_acc"][4] = 1.0                 # seq 2: uniform not in [0, 1)
    kw["temperature"][3] = -1.0          # seq 3: temperature (0 would select greedy verification)
    kw["draft"][8, 5] = np.nan           # seq 4: non-finite logit in a pair
    kw["u_acc"][10:12] = 0.9999          # seq 5: force acceptance of both ...
    kw["target"][5 * 3:5 * 3 + 2] = kw["draft"][10:12]  # ... by equal rows
    kw["target"][5 * 3 + 2, 0] = np.inf  # ... and a bad bonus row
    out = orc.verify(**kw)
    assert list(out["seq_err"]) == [0, orc.BAD_TOKEN, orc.BAD_UNIFORM, orc.BAD_TEMP, orc.BAD_LOGIT,
                                     orc.BAD_LOGIT]
    for b in range(1, 6):
        assert out["accepted"][b] == 0 and (out["tokens"][b] == -1).all()
    assert np.isnan(out["kld"][2:10]).all()
    # a non-finite bonus row withholds only the token
    assert np.isfinite(out["kld"][10:12]).all() and np.isfinite(out["kld"][:2]).all()
    # a bad bonus row of a sequence that rejects early is never read
    kw2 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in base.items()}
    kw2["u_acc"][0] = U_MAX
    kw2["draft_tokens"][0] = int(np.argmin(softmax(kw2["target"][0].astype(np.float64)) /
                                           softmax(kw2["draft"][0].astype(np.float64))))
    kw2["target"][2, 3] = np.nan
    out2 = orc.verify(**kw2)
    assert out2["seq_err"][0] == 0 and out2["accepted"][0] == 0
    # inconsistent layout flags every sequence
    kw3 = dict(base)
    kw3["cu_sl"] = base["cu_sl"].copy()
    kw3["cu_sl"][3] += 1
    assert (orc.verify(**kw3)["seq_err"] == orc.BAD_LAYOUT).all()
    # temperatures outside [2^-16, 2^16]
    kw4 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in base.items()}
    kw4["temperature"][:4] = [2.0 ** -17, 2.0 ** -16, 2.0 ** 16, 2.0 ** 17]
    assert list(orc.verify(**kw4)["seq_err"][:4]) == [orc.BAD_TEMP, 0, 0, orc.BAD_TEMP]


# ---------------------------------------------------------------- KLD signal

def _ring(values_oldest_first, W):
    """A full-or-partial ring holding the given values, next write at head."""
    h = np.zeros(W)
    vals = list(values_oldest_first)[-W:] if W > 0 else []
    n = len(vals)
    head = 3 % W
    for i, v in enumerate(vals):
        h[(head - n + i) % W] = v
    return h, head, n


def _signal_one(orc, hist_vals, W, kld_vals, delta=0.85, n_short=10, n_long=30):
    h, head, cnt = _ring(hist_vals, W)
    sl, cu = packed_layout([len(kld_vals)])
    return orc.kld_signal(sl, cu, np.asarray(kld_vals, np.float64), h[None, :], [head], [cnt],
                          n_short=n_short, n_long=n_long, delta=delta)


def test_weighted_variance_delta_one_is_population_variance(orc):
    rng = np.random.default_rng(11)
    vals = list(rng.random(40))
    out = _signal_one(orc, vals[:-1], 32, [vals[-1]], delta=1.0)
    newest = np.array(vals[::-1][:32])
    assert out["var_short"][0] == pytest.approx(np.var(newest[:10]), rel=1e-12)
    assert out["var_long"][0] == pytest.approx(np.var(newest[:30]), rel=1e-12)


def test_weighted_variance_matches_weighted_moments(orc):
    rng = np.random.default_rng(12)
    vals = list(rng.random(20) * 0.3)
    out = _signal_one(orc, vals[:-1], 32, [vals[-1]], delta=0.85)
    newest = np.array(vals[::-1])
    for n, key in ((10, "var_short"), (20, "var_long")):
        w = 0.85 ** np.arange(n)
        m1 = np.average(newest[:n], weights=w)
        m2 = np.average(newest[:n] ** 2, weights=w)
        assert out[key][0] == pytest.approx(m2 - m1 * m1, rel=1e-9, abs=1e-15)


def test_weighted_variance_two_values_closed_form(orc):
    a, b, d = 0.7, 0.2, 0.85
    out = _signal_one(orc, [b], 8, [a], delta=d)
    assert out["var_short"][0] == pytest.approx(d * (a - b) ** 2 / (1 + d) ** 2, rel=1e-13)
    assert out["mu_last"][0] == a


def test_signal_degenerate_windows(orc):
    out = _signal_one(orc, [], 8, [0.4])                    # one entry
    assert out["var_short"][0] == 0.0 and out["var_long"][0] == 0.0 and out["wvir"][0] == 0.0
    out = _signal_one(orc, [0.25] * 20, 32, [0.25, 0.25])   # constant history
    assert out["var_long"][0] == 0.0 and out["wvir"][0] == 0.0
    out = _signal_one(orc, [], 8, [])                      # nothing verified, empty ring
    assert out["mu_last"][0] == 0.0 and out["sf"][0] == 0.0 and out["count"][0] == 0
    out = _signal_one(orc, [0.1, 0.3], 8, [])              # nothing verified: newest stands in
    assert out["mu_last"][0] == 0.3 and out["count"][0] == 2


def test_signal_push_and_window_sizes(orc):
    W = 12
    vals = list(np.linspace(0.1, 1.2, 12))
    out = _signal_one(orc, vals, W, [0.5, 0.7, 0.9], delta=1.0)
    assert out["mu_last"][0] == pytest.approx(0.7, rel=1e-15)  # mean over all SL positions
    assert out["count"][0] == W and out["head"][0] == (3 + 1) % W
    newest = np.array([0.7] + vals[::-1][:W - 1])
    assert out["var_short"][0] == pytest.approx(np.var(newest[:10]), rel=1e-12)
    assert out["var_long"][0] == pytest.approx(np.var(newest[:W]), rel=1e-12)  # n_long capped by W


def test_scale_factor_closed_form(orc):
    out = _signal_one(orc, [0.1] * 5, 8, [math.log(2.0) / 2] * 3)
    assert out["sf"][0] == pytest.approx(1.0, rel=1e-14)
    out = _signal_one(orc, [0.1] * 5, 8, [0.0, 0.0])
    assert out["sf"][0] == 0.0


def test_wvir_is_ratio_of_window_variances(orc):
    rng = np.random.default_rng(13)
    vals = list(rng.random(31))
    out = _signal_one(orc, vals[:-1], 32, [vals[-1]])
    assert out["wvir"][0] == pytest.approx(out["var_short"][0] / out["var_long"][0], rel=1e-14)


def test_wvir_small_variances_closed_form(orc):
    """Eq. 4 has no guard term: with window variances near 1e-6 WVIR is still
    their plain ratio.  Newest first a, a + 2e-3, a - 1e-3 with delta = 1 and
    windows of 2 and 3: Var_s = (2e-3)^2 / 4 = 1e-6 and Var_l = 42/27 * 1e-6
    (population variance of 0, 2e-3, -1e-3), so WVIR = 27/42."""
    a = 0.1
    out = _signal_one(orc, [a - 1e-3, a + 2e-3], 8, [a], delta=1.0, n_short=2, n_long=3)
    assert out["var_short"][0] == pytest.approx(1e-6, rel=1e-9)
    assert out["var_long"][0] == pytest.approx(42.0 / 27.0 * 1e-6, rel=1e-9)
    assert out["wvir"][0] == pytest.approx(27.0 / 42.0, rel=1e-9)


def test_wvir_constant_window_is_zero_and_eps_must_be_positive(orc):
    # a constant long window (and so a constant short one): variances exactly 0, WVIR = 0
    out = _signal_one(orc, [0.3] * 40, 32, [0.3])
    assert out["var_short"][0] == 0.0 and out["var_long"][0] == 0.0 and out["wvir"][0] == 0.0
    h, head, cnt = _ring([0.3] * 8, 8)
    sl, cu = packed_layout([1])
    with pytest.raises(ValueError):
        orc.kld_signal(sl, cu, np.array([0.3]), h[None, :], [head], [cnt], eps=0.0)


# ---------------------------------------------------------------- SL rule and cap

def test_sl_rule_closed_forms(orc):
    out = orc.next_sl(sf=[0.0, 1.0, 2.0, 0.5, 0.25], wvir=[3.0, 1.0, 1.0, 1.0, 2.0],
                      sl_max=[8.0] * 5, sl_min=2.0, sl_hi=8)
    np.testing.assert_allclose(out["sl_hat"], [8.0, 2.0, 2.0, 5.0, 5.0])
    assert out["sl_cap"] == pytest.approx(22.0 / 5)
    np.testing.assert_array_equal(out["sl_next"], [4, 2, 2, 4, 4])


def test_sl_cap_minimises_mse(orc):
    rng = np.random.default_rng(14)
    sf, wv = rng.random(50) * 0.8, rng.random(50) * 1.5
    out = orc.next_sl(sf, wv, np.full(50, 8.0))
    hat = out["sl_hat"]
    best = minimize_scalar(lambda c: np.mean((c - hat) ** 2), bounds=(0, 10), method="bounded",
                           options={"xatol": 1e-10})
    assert out["sl_cap"] == pytest.approx(best.x, abs=1e-7)
    assert out["sl_cap"] <= hat.max()


def test_sl_rounding_and_errors(orc):
    # SL_hat = 4.5 exactly (pen = 7/12) rounds half up; a NaN input is left out of the cap
    out = orc.next_sl(sf=[7.0 / 12.0, 0.0, np.nan], wvir=[1.0, 0.0, 1.0], sl_max=[8.0, 8.0, 8.0])
    assert out["sl_hat"][0] == pytest.approx(4.5, abs=1e-15)
    assert out["sl_cap"] == pytest.approx((out["sl_hat"][0] + 8.0) / 2)
    assert list(out["sl_next"]) == [5 if out["sl_hat"][0] >= 4.5 else 4, 6, 2]
    assert out["seq_err"][2] == orc.BAD_SIGNAL
    out = orc.next_sl(sf=[0.0], wvir=[0.0], sl_max=[16.0], sl_hi=8)
    assert out["sl_next"][0] == 8   # clamped to the next step's budget


def test_calibration_eq1(orc):
    got = orc.calibrate_sl_max([3, 5, 2], [0.1, 0.3, 0.2])
    assert got == pytest.approx(5.0 * (1.0 + 0.2 / (0.3 + 1e-6)), rel=1e-14)


def test_sl_tie_analysis(orc):
    hat = np.array([4.5, 4.2, 7.0, 3.499995])
    err = np.zeros(4, np.uint32)
    tie = orc.sl_round_ties(hat, np.zeros(4), err, sl_min=2.0, sl_hi=8, tau=1e-5)
    # cap = 4.79999875: x = [4.5, 4.2, 4.8, 3.499995]
    np.testing.assert_array_equal(tie, [1, 0, 0, 1])
    tie = orc.sl_round_ties(hat, np.array([0.0, 0.31, 0.0, 0.0]), err, sl_hi=8, tau=1e-5)
    assert tie[1] == 1
    # spread from a perturbed history: zero when rho = 0
    h, head, cnt = _ring(list(np.linspace(0.01, 0.3, 20)), 32)
    hat2, dh = orc.sl_hat_spread(h[None, :], [head], [cnt], [8.0], [0], rho=0.0)
    assert dh[0] == 0.0
    hat3, dh3 = orc.sl_hat_spread(h[None, :], [head], [cnt], [8.0], [0], rho=1e-4)
    assert hat3[0] == hat2[0] and dh3[0] > 0.0


# ---------------------------------------------------------------------------
# greedy verification (T_b = 0; the temperature-0.0 setting of Sec. 4.2 and
# Table 3(a))
# ---------------------------------------------------------------------------

def _greedy_batch(rng, sls, V, gap=3.0):
    """Random rows whose maxima are unique by at least `gap`."""
    kw = _random_batch(rng, sls, V, T=0.0)
    for rows in (kw["target"], kw["draft"]):
        for r in range(rows.shape[0]):
            rows[r, rng.integers(0, V)] = rows[r].max() + gap
    return kw


def test_greedy_accepts_the_argmax_prefix_and_emits_the_argmax(orc):
    rng = np.random.default_rng(41)
    sls = [4, 3, 2, 0]
    V = 30
    kw = _greedy_batch(rng, sls, V)
    cu = kw["cu_sl"]
    am = lambda r: int(np.argmax(kw["target"][r]))
    # seq 0 accepts 2 drafts, seq 1 all 3, seq 2 none, seq 3 drafted nothing
    for b, acc in ((0, 2), (1, 3), (2, 0)):
        for j in range(sls[b]):
            t = am(cu[b] + b + j)
            kw["draft_tokens"][cu[b] + j] = t if j < acc else (t + 1) % V
    out = orc.verify(**kw)
    assert list(out["seq_err"]) == [0, 0, 0, 0]
    for b, acc in ((0, 2), (1, 3), (2, 0), (3, 0)):
        assert out["accepted"][b] == acc
        toks = out["tokens"][b]
        assert list(toks[:acc]) == list(kw["draft_tokens"][cu[b]: cu[b] + acc])
        assert toks[acc] == am(cu[b] + b + acc)  # the first rejected row, or the bonus row
        assert (toks[acc + 1:] == -1).all()


def test_greedy_ties_take_the_smallest_token(orc):
    rng = np.random.default_rng(42)
    V = 20
    kw = _random_batch(rng, [1, 1], V, T=0.0)
    for r in range(kw["target"].shape[0]):
        m = kw["target"][r].max() + 1.0
        kw["target"][r, [3, 7, 11]] = m  # three equal maxima
    kw["draft_tokens"][:] = [7, 3]       # seq 0 drafts a tied maximum that is not the smallest
    out = orc.verify(**kw)
    assert list(out["accepted"]) == [0, 1]
    assert out["tokens"][0][0] == 3 and list(out["tokens"][1][:2]) == [3, 3]


def test_greedy_is_the_zero_temperature_limit_of_sampling(orc):
    """With unique maxima and drafts drawn from q (at T -> 0: the draft row's
    argmax), sampling at T = 2^-16 accepts exactly the drafts that are the
    target argmax and draws the target argmax, whatever the uniforms."""
    rng = np.random.default_rng(43)
    sls = [3, 1, 4, 2, 0, 5]
    V = 40
    kw = _random_batch(rng, sls, V, T=0.0)
    cu = kw["cu_sl"]
    tgt, dft = kw["target"], kw["draft"]
    for r in range(tgt.shape[0]):
        tgt[r, rng.integers(0, V)] = tgt[r].max() + 3.0
    for b, s in enumerate(sls):
        acc = int(rng.integers(0, s + 1))
        for j in range(s):
            t = int(np.argmax(tgt[cu[b] + b + j]))
            x = t if j < acc else int((t + 1 + rng.integers(0, V - 1)) % V)  # x != t after the prefix
            dft[cu[b] + j, x] = max(dft[cu[b] + j].max(), tgt[cu[b] + b + j].max()) + 3.0
            kw["draft_tokens"][cu[b] + j] = x
    greedy = orc.verify(**kw)
    cold = dict(kw, temperature=np.full(len(sls), 2.0 ** -16, np.float32))
    for trial in range(4):
        cold["u_acc"] = rng.random(len(kw["u_acc"])).astype(np.float32)
        cold["u_res"] = rng.random(len(sls)).astype(np.float32)
        out = orc.verify(**cold)
        assert np.array_equal(out["accepted"], greedy["accepted"])
        assert np.array_equal(out["tokens"], greedy["tokens"])


def test_greedy_kld_is_taken_at_unit_temperature_and_uniforms_are_unused(orc):
    rng = np.random.default_rng(44)
    sls = [2, 3]
    kw = _greedy_batch(rng, sls, 25)
    kw["u_acc"][:] = 1.5   # outside [0, 1): irrelevant for greedy sequences
    kw["u_res"][:] = -1.0
    g = orc.verify(**kw)
    assert list(g["seq_err"]) == [0, 0]
    unit = orc.verify(**dict(kw, temperature=np.ones(2, np.float32),
                             u_acc=np.zeros(5, np.float32), u_res=np.zeros(2, np.float32)))
    np.testing.assert_array_equal(g["kld"], unit["kld"])


# ---------------------------------------------------------------------------
# draft entropy H(q) (the comparison signal of Sec. 4.2, Table 2)
# ---------------------------------------------------------------------------

def test_draft_entropy_closed_forms(orc):
    V = 64
    sls = [3, 2]
    rng = np.random.default_rng(61)
    kw = _random_batch(rng, sls, V, T=1.0)
    kw["draft"][0] = 0.0                         # uniform: ln V
    kw["draft"][1] = 0.0
    kw["draft"][1, 5] = 200.0                    # one-hot: 0
    kw["draft"][2, :2] = [np.log(3.0), 0.0]      # two tokens with q = 3/4, 1/4: the binary entropy
    kw["draft"][2, 2:] = -1e4
    out = orc.verify(**kw)
    np.testing.assert_allclose(out["entropy"][0], np.log(V), rtol=1e-14)
    assert 0.0 <= out["entropy"][1] < 1e-80
    p3 = 1.0 / (1.0 + np.exp(-np.float64(np.float32(np.log(3.0)))))  # q = (3/4, 1/4) up to fp32 rounding of ln 3
    np.testing.assert_allclose(out["entropy"][2], -(p3 * np.log(p3) + (1 - p3) * np.log(1 - p3)), rtol=1e-12)
    for n in range(3, 5):  # random rows: the textbook definition
        q = softmax(kw["draft"][n].astype(np.float64))
        np.testing.assert_allclose(out["entropy"][n], entropy(q), rtol=1e-12)


def test_draft_entropy_is_taken_on_the_tempered_distribution(orc):
    rng = np.random.default_rng(62)
    kw = _random_batch(rng, [2, 2], 30, T=1.0)
    kw["temperature"] = np.array([0.5, 2.0], np.float32)
    out = orc.verify(**kw)
    cu = kw["cu_sl"]
    for b, T in enumerate([0.5, 2.0]):
        for j in range(2):
            q = softmax(kw["draft"][cu[b] + j].astype(np.float64) / T)
            np.testing.assert_allclose(out["entropy"][cu[b] + j], entropy(q), rtol=1e-12)
    g = orc.verify(**dict(kw, temperature=np.zeros(2, np.float32)))  # greedy: at T = 1
    for n in range(4):
        np.testing.assert_allclose(g["entropy"][n], entropy(softmax(kw["draft"][n].astype(np.float64))),
                                   rtol=1e-12)


# ---------------------------------------------------------------------------
# token budget of the policy interface (Sec. 3.2)
# ---------------------------------------------------------------------------

def test_budget_bounds_the_next_length(orc):
    rng = np.random.default_rng(63)
    B = 12
    sf = rng.uniform(0.0, 0.3, B)
    wv = rng.uniform(0.0, 2.0, B)
    mx = np.full(B, 8.0)
    free = orc.next_sl(sf, wv, mx, 2.0, 8)
    same = orc.next_sl(sf, wv, mx, 2.0, 8, budget=np.full(B, 10 ** 6, np.int32))
    assert np.array_equal(free["sl_next"], same["sl_next"])
    budget = np.array([0, 1, 2, 3, 4, 5, 6, 7, 8, 9, -3, 100], np.int32)
    got = orc.next_sl(sf, wv, mx, 2.0, 8, budget=budget)
    assert np.array_equal(got["sl_next"], np.minimum(free["sl_next"], np.maximum(budget - 1, 0)))
    assert got["sl_cap"] == free["sl_cap"]  # the cap is taken before the budget
