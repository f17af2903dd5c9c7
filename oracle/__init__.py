"""CPU oracle for the DSDE verification step -- TEST INFRASTRUCTURE ONLY.

Thin ctypes wrapper around ``dsde_oracle.c`` (plain fp64 C, see its header
for what each function follows in the paper).  Only the tests, the smoke
check and the benchmark's CPU-baseline leg may import this package; the HIP
library never does.

Arrays are numpy arrays on the host.  Logits are passed as ``uint16`` (bf16
bit patterns) or ``float32``.
"""
import ctypes
import os

import numpy as np

from .build_oracle import LIB, build

_lib = None

# per-sequence error bits reported by the oracle
BAD_LAYOUT, BAD_TOKEN, BAD_LOGIT, BAD_TEMP, BAD_UNIFORM, BAD_SIGNAL, BAD_STATE = 1, 2, 4, 8, 16, 32, 64
TIE_BAND = 1e-6


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.environ.get("DSDE_ORACLE_LIB", LIB)  # a mutated build, for the mutation tests
    if path == LIB and not os.path.exists(LIB):
        build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.oracle_verify.argtypes = [P, P, i32, i64, i32, i32, i64, P, P, P, P, P, P, i32,
                                  P, P, P, P, P, P, P, P, P, i32]
    lib.oracle_verify.restype = i32
    lib.oracle_kld_signal.argtypes = [i32, i64, P, P, P, P, P, P, i32, i32, i32, f64, f64,
                                      P, P, P, P, P, P]
    lib.oracle_kld_signal.restype = i32
    lib.oracle_next_sl.argtypes = [i32, P, P, P, f64, i32, P, P, P, P, P]
    lib.oracle_next_sl.restype = i32
    lib.oracle_calibrate_sl_max.argtypes = [i32, P, i64, P, f64]
    lib.oracle_calibrate_sl_max.restype = f64
    lib.oracle_signal_spread.argtypes = [i32, P, P, P, i32, P, i32, i32, f64, f64, f64, f64, P, P, P, P, P, P,
                                         P]
    lib.oracle_signal_spread.restype = i32
    lib.oracle_sl_round_ties.argtypes = [i32, P, P, P, f64, i32, f64, P]
    lib.oracle_sl_round_ties.restype = i32
    _lib = lib
    return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def verify(target, draft, V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max,
           pad_id=-1, n_threads=1):
    """Speculative verification of one step (see ``oracle_verify``).

    ``target``: [N+B, V] and ``draft``: [N, V] logits (uint16 bf16 bits or float32).
    Returns a dict of numpy arrays: accepted [B], tokens [B, k_max+1], kld [N] (fp64),
    lse [N, 2] (fp64), entropy [N] (H(q) in nats, fp64), seq_err [B], acc_tie [B],
    cdf_tie [B], sample_mass [B].
    """
    lib = _load()
    if target.dtype == np.uint16:
        dtype = 1
    elif target.dtype == np.float32:
        dtype = 0
    else:
        raise TypeError("logits must be uint16 (bf16 bits) or float32")
    assert draft.dtype == target.dtype
    sl_a, sl_p = _c(sl, np.int32)
    cu_a, cu_p = _c(cu_sl, np.int32)
    B = sl_a.shape[0]
    N = int(draft.size // V) if V > 0 else 0
    t_a, t_p = _c(target, target.dtype)
    d_a, d_p = _c(draft, draft.dtype)
    tok_a, tok_p = _c(draft_tokens, np.int32)
    T_a, T_p = _c(temperature, np.float32)
    ua_a, ua_p = _c(u_acc, np.float32)
    ur_a, ur_p = _c(u_res, np.float32)
    out = {
        "accepted": np.zeros(B, np.int32),
        "tokens": np.zeros((B, k_max + 1), np.int32),
        "kld": np.full(max(N, 1), np.nan, np.float64)[:N],
        "lse": np.full((max(N, 1), 2), np.nan, np.float64)[:N],
        "entropy": np.full(max(N, 1), np.nan, np.float64)[:N],
        "seq_err": np.zeros(B, np.uint32),
        "acc_tie": np.zeros(B, np.int32),
        "cdf_tie": np.zeros(B, np.int32),
        "sample_mass": np.zeros(B, np.float64),
    }
    ptr = {k: v.ctypes.data_as(ctypes.c_void_p) for k, v in out.items()}
    rc = lib.oracle_verify(t_p, d_p, dtype, V, B, k_max, N, sl_p, cu_p, tok_p, T_p, ua_p, ur_p,
                           pad_id, ptr["accepted"], ptr["tokens"], ptr["kld"], ptr["lse"], ptr["entropy"],
                           ptr["seq_err"], ptr["acc_tie"], ptr["cdf_tie"], ptr["sample_mass"],
                           n_threads)
    if rc != 0:
        raise ValueError("oracle_verify rejected its arguments")
    return out


def kld_signal(sl, cu_sl, kld, hist, head, count, n_short=10, n_long=30, delta=0.85, eps=1e-6):
    """Signal update of Sec. 3.1.2 (see ``oracle_kld_signal``).

    ``hist`` [B, W], ``head`` [B], ``count`` [B] are copied, updated and returned.
    """
    lib = _load()
    sl_a, sl_p = _c(sl, np.int32)
    cu_a, cu_p = _c(cu_sl, np.int32)
    B = sl_a.shape[0]
    kld_a, kld_p = _c(kld, np.float64)
    N = kld_a.shape[0]
    hist = np.array(hist, dtype=np.float64, copy=True, order="C")
    W = hist.shape[1]
    head = np.array(head, dtype=np.int32, copy=True)
    count = np.array(count, dtype=np.int32, copy=True)
    out = {k: np.zeros(B, np.float64) for k in ("mu_last", "var_short", "var_long", "wvir", "sf")}
    out["seq_err"] = np.zeros(B, np.uint32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    rc = lib.oracle_kld_signal(B, N, sl_p, cu_p, kld_p, P(hist), P(head), P(count), W, n_short,
                               n_long, delta, eps, P(out["mu_last"]), P(out["var_short"]),
                               P(out["var_long"]), P(out["wvir"]), P(out["sf"]), P(out["seq_err"]))
    if rc != 0:
        raise ValueError("oracle_kld_signal rejected its arguments")
    out.update(hist=hist, head=head, count=count)
    return out


def next_sl(sf, wvir, sl_max, sl_min=2.0, sl_hi=8, budget=None):
    """SL rule (Eqs. 2, 8) and batch cap (Eqs. 9-11) (see ``oracle_next_sl``);
    ``budget`` [B] int32 (optional): tokens each sequence may still emit."""
    lib = _load()
    sf_a, sf_p = _c(sf, np.float64)
    wv_a, wv_p = _c(wvir, np.float64)
    mx_a, mx_p = _c(sl_max, np.float64)
    B = sf_a.shape[0]
    hat = np.zeros(B, np.float64)
    cap = np.zeros(1, np.float64)
    nxt = np.zeros(B, np.int32)
    err = np.zeros(B, np.uint32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    bud_p = None
    if budget is not None:
        bud_a, bud_p = _c(budget, np.int32)
    rc = lib.oracle_next_sl(B, sf_p, wv_p, mx_p, sl_min, sl_hi, bud_p, P(hat), P(cap), P(nxt), P(err))
    if rc != 0:
        raise ValueError("oracle_next_sl rejected its arguments")
    return {"sl_hat": hat, "sl_cap": float(cap[0]), "sl_next": nxt, "seq_err": err}


def calibrate_sl_max(accepted_per_step, kld_values, eps=1e-6):
    """Eq. 1: SL_max from the calibration steps' accepted counts and KLD values."""
    lib = _load()
    a_a, a_p = _c(accepted_per_step, np.int32)
    k_a, k_p = _c(kld_values, np.float64)
    return float(lib.oracle_calibrate_sl_max(a_a.shape[0], a_p, k_a.shape[0], k_p, eps))


def signal_spread(hist, head, count, sl_max, seq_err, n_short=10, n_long=30, delta=0.85, eps=1e-6,
                  sl_min=2.0, rho=1e-4):
    """First-order spreads of var_short, var_long, wvir, sf and SL_hat under a relative
    uncertainty ``rho`` on every history entry (post-step rings).  Returns a dict with
    ``sl_hat`` and the spreads ``d_var_short``, ``d_var_long``, ``d_wvir``, ``d_sf``,
    ``d_sl_hat``."""
    lib = _load()
    h_a, h_p = _c(hist, np.float64)
    B, W = h_a.shape
    hd_a, hd_p = _c(head, np.int32)
    c_a, c_p = _c(count, np.int32)
    mx_a, mx_p = _c(sl_max, np.float64)
    e_a, e_p = _c(seq_err, np.uint32)
    out = {k: np.zeros(B, np.float64) for k in ("sl_hat", "d_sl_hat", "d_var_short", "d_var_long", "d_wvir",
                                                 "d_sf")}
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    lib.oracle_signal_spread(B, h_p, hd_p, c_p, W, mx_p, n_short, n_long, delta, eps, sl_min, rho, e_p,
                             P(out["sl_hat"]), P(out["d_sl_hat"]), P(out["d_var_short"]), P(out["d_var_long"]),
                             P(out["d_wvir"]), P(out["d_sf"]))
    return out


def sl_hat_spread(hist, head, count, sl_max, seq_err, rho=1e-4, **kw):
    """SL_hat and its first-order spread (see ``signal_spread``)."""
    o = signal_spread(hist, head, count, sl_max, seq_err, rho=rho, **kw)
    return o["sl_hat"], o["d_sl_hat"]


def sl_round_ties(hat, dhat, seq_err, sl_min=2.0, sl_hi=8, tau=1e-5):
    """Flags SL decisions whose rounding could flip within the given spreads."""
    lib = _load()
    h_a, h_p = _c(hat, np.float64)
    d_a, d_p = _c(dhat, np.float64)
    e_a, e_p = _c(seq_err, np.uint32)
    B = h_a.shape[0]
    tie = np.zeros(B, np.int32)
    lib.oracle_sl_round_ties(B, h_p, d_p, e_p, sl_min, sl_hi, tau, tie.ctypes.data_as(ctypes.c_void_p))
    return tie
