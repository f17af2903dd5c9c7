"""DSDE speculative-verification hot path on MI355X (gfx950).

Python binding of libdsde.so (declared in include/dsde.h): the same entry
points, taking torch tensors that already live on the GPU.  This module only
checks shapes/dtypes and marshals pointers and the current HIP stream; every
step of the computation runs in the library's HIP kernels.  There is no CPU
fallback: if the library is missing, ``load`` raises.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdsde.so")

OK, INVALID_ARG, WORKSPACE_TOO_SMALL, DEVICE_ERROR = 0, 1, 2, 3
FP32, BF16 = 0, 1
ERR_LAYOUT, ERR_TOKEN, ERR_LOGIT, ERR_TEMP, ERR_UNIFORM, ERR_SIGNAL, ERR_STATE = 1, 2, 4, 8, 16, 32, 64
MAX_K = 63
STATIC_SCRATCH_BYTES = 16 << 20  # DSDE_STATIC_SCRATCH_BYTES: the scratch array of dsde_step_static
EXPORTS = ("dsde_abi_version", "dsde_status_string", "dsde_verify_workspace_bytes", "dsde_verify",
           "dsde_step", "dsde_step_static", "dsde_kld_signal", "dsde_next_sl", "dsde_calibration_update", "dsde_calibrate_sl_max",
           "dsde_set_profile_events", "dsde_stream_read", "dsde_shard_workspace_bytes", "dsde_shard_stats",
           "dsde_shard_accept", "dsde_shard_accept_step", "dsde_shard_draw_mass", "dsde_shard_draw_pick")
# sizes of the records the vocabulary-shard calls exchange (dsde_shard_partial,
# dsde_draw_job, dsde_shard_mass); kept as raw bytes on the Python side
SHARD_PARTIAL_BYTES, DRAW_JOB_BYTES, SHARD_MASS_BYTES = 64, 44, 32

_lib = None


class DsdeError(RuntimeError):
    pass


def load(path: str = LIB_PATH):
    """Load libdsde.so (built by ``build_lib.build``); raises when it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise DsdeError(f"{path} is missing: build it with __graft_entry__.build() "
                        "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    P, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    lib.dsde_abi_version.restype = i32
    lib.dsde_abi_version.argtypes = []
    lib.dsde_status_string.restype = ctypes.c_char_p
    lib.dsde_status_string.argtypes = [i32]
    lib.dsde_verify_workspace_bytes.restype = sz
    lib.dsde_verify_workspace_bytes.argtypes = [i32, i64, i64, i32]
    lib.dsde_verify.restype = i32
    lib.dsde_verify.argtypes = [P, P, i32, i64, i32, i64, i32, P, P, P, P, P, P, i32, P, P, P, P, P, P, P, sz, P]
    lib.dsde_step.restype = i32
    lib.dsde_step.argtypes = [P, P, i32, i64, i32, i64, i32, P, P, P, P, P, P, i32, P, P, P, P, P,
                              P, P, P, i32, i32, i32, f32, f32, P, P, P, P, P,
                              P, f32, i32, P, P, P, P, P, P, sz, P]
    lib.dsde_step_static.restype = i32
    lib.dsde_step_static.argtypes = [P, P, i32, i64, i32, i64, i32, P, P, P, P, P, P, i32, P, P, P, P, P,
                                     P, P, P, i32, i32, i32, f32, f32, P, P, P, P, P,
                                     P, f32, i32, P, P, P, P, P, P]
    lib.dsde_kld_signal.restype = i32
    lib.dsde_kld_signal.argtypes = [i32, i64, P, P, P, P, P, P, i32, i32, i32, f32, f32, P, P, P, P, P, P, P]
    lib.dsde_next_sl.restype = i32
    lib.dsde_next_sl.argtypes = [i32, P, P, P, f32, i32, P, P, P, P, P, P]
    lib.dsde_calibration_update.restype = i32
    lib.dsde_calibration_update.argtypes = [i32, i64, P, P, P, P, P, P, P, P, P, P]
    lib.dsde_calibrate_sl_max.restype = i32
    lib.dsde_calibrate_sl_max.argtypes = [i32, P, P, P, P, f32, i32, P, P]
    lib.dsde_set_profile_events.restype = i32
    lib.dsde_set_profile_events.argtypes = [P, P]
    lib.dsde_stream_read.restype = i32
    lib.dsde_stream_read.argtypes = [P, i64, P, P]
    lib.dsde_shard_workspace_bytes.restype = sz
    lib.dsde_shard_workspace_bytes.argtypes = [i32, i64, i64, i32]
    lib.dsde_shard_stats.restype = i32
    lib.dsde_shard_stats.argtypes = [P, P, i32, i64, i64, i64, i32, i64, i32, P, P, P, P, P, P, P, sz, P]
    lib.dsde_shard_accept.restype = i32
    lib.dsde_shard_accept.argtypes = [i32, P, i64, i32, i64, i32, P, P, P, P, P, P, i32, P, P, P, P, P, P, P, P]
    lib.dsde_shard_accept_step.restype = i32
    lib.dsde_shard_accept_step.argtypes = [i32, P, i64, i32, i64, i32, P, P, P, P, P, P, i32, P, P, P, P, P, P,
                                           P, P, P, i32, i32, i32, f32, f32, P, P, P, P, P,
                                           P, f32, i32, P, P, P, P, P, P]
    lib.dsde_shard_draw_mass.restype = i32
    lib.dsde_shard_draw_mass.argtypes = [P, P, i32, i64, i64, i32, i64, i32, P, P, P, P, sz, P]
    lib.dsde_shard_draw_pick.restype = i32
    lib.dsde_shard_draw_pick.argtypes = [i32, i32, P, P, P, i32, i64, i64, i32, i64, i32, P, i32, P, P, P, P, P,
                                         sz, P]
    _lib = lib
    return lib


def _check(rc):
    if rc != OK:
        raise DsdeError(f"libdsde: {load().dsde_status_string(rc).decode()} (status {rc})")


def _ptr(t, dtype=None, n=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise DsdeError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise DsdeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise DsdeError(f"{name} must be contiguous")
    if n is not None and t.numel() < n:
        raise DsdeError(f"{name} has {t.numel()} elements, needs {n}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def workspace_bytes(B, N, V, k_max):
    return int(load().dsde_verify_workspace_bytes(B, N, V, k_max))


def new_workspace(B, N, V, k_max, device="cuda"):
    n = workspace_bytes(B, N, V, k_max)
    if n == 0:
        raise DsdeError("invalid sizes for the verify workspace")
    return torch.empty(n, dtype=torch.uint8, device=device)


def verify(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, pad_id=-1,
           out=None, workspace=None, row_lse=None, draft_entropy=False, stream=None):
    """``dsde_verify`` on torch tensors.  Returns a dict with accepted, tokens, kld,
    seq_err (and draft_entropy when asked for); pass ``out`` (a dict with those
    keys) to reuse output buffers."""
    lib = load()
    dt = _logits_dtype(target)
    V = int(target.shape[1])
    B = int(sl.shape[0])
    N = int(draft.shape[0]) if draft is not None else 0
    dev = target.device
    if draft is not None and (draft.dtype != target.dtype or (N > 0 and int(draft.shape[1]) != V)):
        raise DsdeError("draft logits must match the target's dtype and vocabulary")
    if int(target.shape[0]) != N + B:
        raise DsdeError(f"target has {target.shape[0]} rows, expected N + B = {N + B}")
    if out is None:
        out = {"accepted": torch.empty(B, dtype=torch.int32, device=dev),
               "tokens": torch.empty((B, k_max + 1), dtype=torch.int32, device=dev),
               "kld": torch.empty(max(N, 1), dtype=torch.float32, device=dev)[:N],
               "seq_err": torch.empty(B, dtype=torch.int32, device=dev)}
    if draft_entropy and "draft_entropy" not in out:
        out["draft_entropy"] = torch.empty(max(N, 1), dtype=torch.float32, device=dev)[:N]
    ent = out.get("draft_entropy") if draft_entropy else None
    if workspace is None:
        workspace = new_workspace(B, N, V, k_max, device=dev)
    rc = lib.dsde_verify(
        _ptr(target, name="target"), _ptr(draft, name="draft") if N > 0 else None, dt, V, B, N, k_max,
        _ptr(sl, torch.int32, B, "sl"), _ptr(cu_sl, torch.int32, B + 1, "cu_sl"),
        _ptr(draft_tokens, torch.int32, N, "draft_tokens") if N > 0 else None,
        _ptr(temperature, torch.float32, B, "temperature"),
        _ptr(u_acc, torch.float32, N, "u_acc") if N > 0 else None,
        _ptr(u_res, torch.float32, B, "u_res"), int(pad_id),
        _ptr(out["accepted"], torch.int32, B, "accepted"),
        _ptr(out["tokens"], torch.int32, B * (k_max + 1), "tokens"),
        _ptr(out["kld"], torch.float32, N, "kld") if N > 0 else None,
        _ptr(out["seq_err"], None, B, "seq_err"),
        _ptr(row_lse, torch.float64, 2 * N, "row_lse") if row_lse is not None else None,
        _ptr(ent, torch.float32, N, "draft_entropy") if ent is not None and N > 0 else None,
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(), _stream(stream))
    _check(rc)
    return out


def _logits_dtype(target):
    if target.dtype == torch.bfloat16:
        return BF16
    if target.dtype == torch.float32:
        return FP32
    raise DsdeError("logits must be bfloat16 or float32")


def _step_args(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, hist, head, count,
               sl_max, n_short, n_long, delta, eps, sl_min, sl_hi, pad_id, out, row_lse, draft_entropy, budget):
    """Marshalled arguments of dsde_step up to seq_err (shared with dsde_step_static), and the outputs."""
    dt = _logits_dtype(target)
    V = int(target.shape[1])
    B = int(sl.shape[0])
    N = int(draft.shape[0]) if draft is not None else 0
    W = int(hist.shape[1])
    sl_hi = k_max if sl_hi is None else sl_hi
    dev = target.device
    if int(target.shape[0]) != N + B:
        raise DsdeError(f"target has {target.shape[0]} rows, expected N + B = {N + B}")
    if out is None:
        out = {"accepted": torch.empty(B, dtype=torch.int32, device=dev),
               "tokens": torch.empty((B, k_max + 1), dtype=torch.int32, device=dev),
               "kld": torch.empty(max(N, 1), dtype=torch.float32, device=dev)[:N],
               "seq_err": torch.empty(B, dtype=torch.int32, device=dev),
               "sl_cap": torch.empty(1, dtype=torch.float32, device=dev),
               "sl_next": torch.empty(B, dtype=torch.int32, device=dev)}
        for k in ("mu_last", "var_short", "var_long", "wvir", "sf", "sl_hat"):
            out[k] = torch.empty(B, dtype=torch.float32, device=dev)
    if draft_entropy and "draft_entropy" not in out:
        out["draft_entropy"] = torch.empty(max(N, 1), dtype=torch.float32, device=dev)[:N]
    ent = out.get("draft_entropy") if draft_entropy else None
    f32 = torch.float32
    args = [
        _ptr(target, name="target"), _ptr(draft, name="draft") if N > 0 else None, dt, V, B, N, k_max,
        _ptr(sl, torch.int32, B, "sl"), _ptr(cu_sl, torch.int32, B + 1, "cu_sl"),
        _ptr(draft_tokens, torch.int32, N, "draft_tokens") if N > 0 else None,
        _ptr(temperature, f32, B, "temperature"), _ptr(u_acc, f32, N, "u_acc") if N > 0 else None,
        _ptr(u_res, f32, B, "u_res"), int(pad_id),
        _ptr(out["accepted"], torch.int32, B), _ptr(out["tokens"], torch.int32, B * (k_max + 1)),
        _ptr(out["kld"], f32, N) if N > 0 else None,
        _ptr(row_lse, torch.float64, 2 * N, "row_lse") if row_lse is not None else None,
        _ptr(ent, f32, N, "draft_entropy") if ent is not None and N > 0 else None,
        _ptr(hist, f32, B * W, "hist"), _ptr(head, torch.int32, B, "head"), _ptr(count, torch.int32, B, "count"),
        W, n_short, n_long, float(delta), float(eps),
        _ptr(out["mu_last"], f32, B), _ptr(out["var_short"], f32, B), _ptr(out["var_long"], f32, B),
        _ptr(out["wvir"], f32, B), _ptr(out["sf"], f32, B), _ptr(sl_max, f32, B, "sl_max"), float(sl_min),
        int(sl_hi), _ptr(budget, torch.int32, B, "budget") if budget is not None else None,
        _ptr(out["sl_hat"], f32, B), _ptr(out["sl_cap"], f32, 1), _ptr(out["sl_next"], torch.int32, B),
        _ptr(out["seq_err"], None, B)]
    return args, out, (B, N, V)


def step(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, hist, head, count,
         sl_max, n_short=10, n_long=30, delta=0.85, eps=1e-6, sl_min=2.0, sl_hi=None, pad_id=-1,
         out=None, workspace=None, row_lse=None, draft_entropy=False, budget=None, stream=None):
    """``dsde_step``: verify + signal update + SL rule in one call.  hist/head/count are
    updated in place; returns a dict of every output (accepted, tokens, kld, mu_last,
    var_short, var_long, wvir, sf, sl_hat, sl_cap, sl_next, seq_err, and draft_entropy
    when asked for).  ``budget`` [B] int32: tokens each sequence may still emit."""
    lib = load()
    args, out, (B, N, V) = _step_args(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max,
                                      hist, head, count, sl_max, n_short, n_long, delta, eps, sl_min, sl_hi, pad_id,
                                      out, row_lse, draft_entropy, budget)
    if workspace is None:
        workspace = new_workspace(B, N, V, k_max, device=target.device)
    rc = lib.dsde_step(*args, _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(), _stream(stream))
    _check(rc)
    return out


def step_static(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, hist, head, count,
                sl_max, n_short=10, n_long=30, delta=0.85, eps=1e-6, sl_min=2.0, sl_hi=None, pad_id=-1,
                out=None, row_lse=None, draft_entropy=False, budget=None, stream=None):
    """``dsde_step_static``: ``step`` without a workspace argument; the library's
    per-device scratch array (STATIC_SCRATCH_BYTES) holds the scratch space, and
    the call allocates no device memory when ``out`` is given.  Calls that may
    overlap on one GPU share that array and must not run concurrently."""
    lib = load()
    args, out, _ = _step_args(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, hist, head,
                              count, sl_max, n_short, n_long, delta, eps, sl_min, sl_hi, pad_id, out, row_lse,
                              draft_entropy, budget)
    _check(lib.dsde_step_static(*args, _stream(stream)))
    return out


def kld_signal(sl, cu_sl, kld, hist, head, count, n_short=10, n_long=30, delta=0.85, eps=1e-6,
               out=None, stream=None):
    """``dsde_kld_signal``: updates hist/head/count in place; returns the outputs."""
    lib = load()
    B = int(sl.shape[0])
    N = int(kld.shape[0])
    W = int(hist.shape[1])
    dev = sl.device
    if out is None:
        out = {k: torch.empty(B, dtype=torch.float32, device=dev)
               for k in ("mu_last", "var_short", "var_long", "wvir", "sf")}
        out["seq_err"] = torch.empty(B, dtype=torch.int32, device=dev)
    rc = lib.dsde_kld_signal(
        B, N, _ptr(sl, torch.int32, B, "sl"), _ptr(cu_sl, torch.int32, B + 1, "cu_sl"),
        _ptr(kld, torch.float32, N, "kld") if N > 0 else None, _ptr(hist, torch.float32, B * W, "hist"),
        _ptr(head, torch.int32, B, "head"), _ptr(count, torch.int32, B, "count"), W, n_short, n_long,
        float(delta), float(eps), _ptr(out["mu_last"], torch.float32, B), _ptr(out["var_short"], torch.float32, B),
        _ptr(out["var_long"], torch.float32, B), _ptr(out["wvir"], torch.float32, B),
        _ptr(out["sf"], torch.float32, B), _ptr(out["seq_err"], None, B), _stream(stream))
    _check(rc)
    return out


def next_sl(sf, wvir, sl_max, sl_min=2.0, sl_hi=8, budget=None, out=None, stream=None):
    """``dsde_next_sl``: SL rule with the batch cap (and the optional per-sequence
    token budget); returns sl_hat, sl_cap, sl_next, seq_err."""
    lib = load()
    B = int(sf.shape[0])
    dev = sf.device
    if out is None:
        out = {"sl_hat": torch.empty(B, dtype=torch.float32, device=dev),
               "sl_cap": torch.empty(1, dtype=torch.float32, device=dev),
               "sl_next": torch.empty(B, dtype=torch.int32, device=dev),
               "seq_err": torch.empty(B, dtype=torch.int32, device=dev)}
    rc = lib.dsde_next_sl(B, _ptr(sf, torch.float32, B, "sf"), _ptr(wvir, torch.float32, B, "wvir"),
                          _ptr(sl_max, torch.float32, B, "sl_max"), float(sl_min), int(sl_hi),
                          _ptr(budget, torch.int32, B, "budget") if budget is not None else None,
                          _ptr(out["sl_hat"], torch.float32, B), _ptr(out["sl_cap"], torch.float32, 1),
                          _ptr(out["sl_next"], torch.int32, B), _ptr(out["seq_err"], None, B), _stream(stream))
    _check(rc)
    return out


def new_calibration_state(B, device="cuda"):
    """Zeroed running statistics of the SL_max calibration (Eq. 1)."""
    return {"a_max": torch.zeros(B, dtype=torch.int32, device=device),
            "kld_sum": torch.zeros(B, dtype=torch.float64, device=device),
            "kld_count": torch.zeros(B, dtype=torch.int64, device=device),
            "kld_max": torch.zeros(B, dtype=torch.float32, device=device)}


def calibration_update(sl, cu_sl, accepted, kld, seq_err, state, stream=None):
    """``dsde_calibration_update``: folds one verification step into ``state``."""
    lib = load()
    B = int(sl.shape[0])
    N = int(kld.shape[0])
    _check(lib.dsde_calibration_update(
        B, N, _ptr(sl, torch.int32, B, "sl"), _ptr(cu_sl, torch.int32, B + 1, "cu_sl"),
        _ptr(accepted, torch.int32, B, "accepted"), _ptr(kld, torch.float32, N, "kld") if N > 0 else None,
        _ptr(seq_err, None, B, "seq_err"), _ptr(state["a_max"], torch.int32, B),
        _ptr(state["kld_sum"], torch.float64, B), _ptr(state["kld_count"], torch.int64, B),
        _ptr(state["kld_max"], torch.float32, B), _stream(stream)))


def calibrate_sl_max(state, eps=1e-6, pooled=False, out=None, stream=None):
    """``dsde_calibrate_sl_max``: Eq. 1 per sequence, or pooled over the batch."""
    lib = load()
    B = int(state["a_max"].shape[0])
    if out is None:
        out = torch.empty(B, dtype=torch.float32, device=state["a_max"].device)
    _check(lib.dsde_calibrate_sl_max(
        B, _ptr(state["a_max"], torch.int32, B), _ptr(state["kld_sum"], torch.float64, B),
        _ptr(state["kld_count"], torch.int64, B), _ptr(state["kld_max"], torch.float32, B), float(eps),
        1 if pooled else 0, _ptr(out, torch.float32, B), _stream(stream)))
    return out


def set_profile_events(start=None, stop=None):
    """Attach HIP events ``start``/``stop`` to the row-statistics kernel of every
    later ``verify``/``step`` call (None, None turns it off).  Each is a
    torch.cuda.Event or a raw hipEvent_t handle (int)."""
    lib = load()

    def handle(ev):
        if ev is None:
            return None
        return ctypes.c_void_p(ev if isinstance(ev, int) else ev.cuda_event)
    _check(lib.dsde_set_profile_events(handle(start), handle(stop)))


def stream_read(buf, out):
    """Streaming-read ceiling probe: reads every byte of the contiguous device
    tensor ``buf`` (one workgroup per 32 KiB) and writes each unit's XOR to
    ``out`` (int32, at least ceil(bytes / 32768) elements) on the current stream."""
    import torch
    lib = load()
    nbytes = buf.numel() * buf.element_size()
    if out.numel() < (nbytes + 32767) // 32768:
        raise DsdeError("stream_read: out holds fewer than one word per 32 KiB")
    _check(lib.dsde_stream_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(out.data_ptr()),
                                ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)))


# ---------------------------------------------------------------------------
# vocabulary-sharded verification (dsde_shard_*): one shard's four calls
# ---------------------------------------------------------------------------

def new_shard_workspace(B, N, V_shard, k_max, device="cuda"):
    n = int(load().dsde_shard_workspace_bytes(B, N, V_shard, k_max))
    if n == 0:
        raise DsdeError("invalid sizes for the shard workspace")
    return torch.empty(n, dtype=torch.uint8, device=device)


def _shard_rows(target, draft, B):
    dt = _logits_dtype(target)
    V_shard = int(target.shape[1])
    N = int(draft.shape[0]) if draft is not None else 0
    if draft is not None and (draft.dtype != target.dtype or (N > 0 and int(draft.shape[1]) != V_shard)):
        raise DsdeError("draft slice must match the target slice's dtype and width")
    if int(target.shape[0]) != N + B:
        raise DsdeError(f"target slice has {target.shape[0]} rows, expected N + B = {N + B}")
    return dt, V_shard, N


def shard_stats(target, draft, v_begin, V, sl, cu_sl, draft_tokens, temperature, k_max, workspace,
                part=None, seq_err=None, stream=None):
    """``dsde_shard_stats`` (call 1) on this shard's slices [rows, V_shard].  Returns
    (part [N, 64] uint8 records, seq_err [B] int32)."""
    lib = load()
    B = int(sl.shape[0])
    dt, V_shard, N = _shard_rows(target, draft, B)
    dev = target.device
    if part is None:
        part = torch.empty((max(N, 1), SHARD_PARTIAL_BYTES), dtype=torch.uint8, device=dev)
    if seq_err is None:
        seq_err = torch.empty(B, dtype=torch.int32, device=dev)
    rc = lib.dsde_shard_stats(
        _ptr(target, name="target"), _ptr(draft, name="draft") if N > 0 else None, dt, V_shard, int(v_begin),
        int(V), B, N, k_max, _ptr(sl, torch.int32, B, "sl"), _ptr(cu_sl, torch.int32, B + 1, "cu_sl"),
        _ptr(draft_tokens, torch.int32, N, "draft_tokens") if N > 0 else None,
        _ptr(temperature, torch.float32, B, "temperature"),
        _ptr(part, torch.uint8, N * SHARD_PARTIAL_BYTES, "part") if N > 0 else None,
        _ptr(seq_err, None, B, "seq_err"), _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(),
        _stream(stream))
    _check(rc)
    return part, seq_err


def _shard_accept_call(parts, V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, seq_err, pad_id,
                       row_lse, draft_entropy, out, stream):
    """Output buffers and the leading ctypes arguments shared by the two call-2 entry points."""
    G = int(parts.shape[0])
    B = int(sl.shape[0])
    N = int(draft_tokens.shape[0]) if draft_tokens is not None else 0
    dev = sl.device
    if N > 0 and (parts.dim() != 3 or int(parts.shape[1]) < N or int(parts.shape[2]) != SHARD_PARTIAL_BYTES):
        raise DsdeError("parts must be [G, N, 64] uint8")
    if out is None:
        out = {"accepted": torch.empty(B, dtype=torch.int32, device=dev),
               "tokens": torch.empty((B, k_max + 1), dtype=torch.int32, device=dev),
               "kld": torch.empty(max(N, 1), dtype=torch.float32, device=dev)[:N],
               "jobs": torch.empty((B, DRAW_JOB_BYTES), dtype=torch.uint8, device=dev)}
    out["seq_err"] = seq_err
    if draft_entropy and "draft_entropy" not in out:
        out["draft_entropy"] = torch.empty(max(N, 1), dtype=torch.float32, device=dev)[:N]
    ent = out.get("draft_entropy") if draft_entropy else None
    if N > 0 and int(parts.shape[1]) != N:
        # the packed copy is made on the call's stream, ahead of the call
        with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
            parts = parts[:, :N].contiguous()
    args = [G, _ptr(parts, torch.uint8, G * N * SHARD_PARTIAL_BYTES, "parts") if N > 0 else None, int(V), B, N,
            k_max, _ptr(sl, torch.int32, B, "sl"), _ptr(cu_sl, torch.int32, B + 1, "cu_sl"),
            _ptr(draft_tokens, torch.int32, N, "draft_tokens") if N > 0 else None,
            _ptr(temperature, torch.float32, B, "temperature"),
            _ptr(u_acc, torch.float32, N, "u_acc") if N > 0 else None, _ptr(u_res, torch.float32, B, "u_res"),
            int(pad_id), _ptr(out["accepted"], torch.int32, B, "accepted"),
            _ptr(out["tokens"], torch.int32, B * (k_max + 1), "tokens"),
            _ptr(out["kld"], torch.float32, N, "kld") if N > 0 else None,
            _ptr(row_lse, torch.float64, 2 * N, "row_lse") if row_lse is not None else None,
            _ptr(ent, torch.float32, N, "draft_entropy") if ent is not None and N > 0 else None,
            _ptr(out["jobs"], torch.uint8, B * DRAW_JOB_BYTES, "jobs")]
    return out, args, parts


def shard_accept(parts, V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, seq_err, pad_id=-1,
                 row_lse=None, draft_entropy=False, out=None, stream=None):
    """``dsde_shard_accept`` (call 2) from the gathered partials parts [G, N, 64]
    (uint8, shard order).  seq_err (call 1's) is updated in place.  Returns a dict
    with accepted, tokens, kld, seq_err, jobs [B, 44] uint8 (and draft_entropy)."""
    lib = load()
    out, args, _keep = _shard_accept_call(parts, V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max,
                                          seq_err, pad_id, row_lse, draft_entropy, out, stream)
    B = int(sl.shape[0])
    _check(lib.dsde_shard_accept(*args, _ptr(seq_err, None, B, "seq_err"), _stream(stream)))
    return out


def shard_accept_step(parts, V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, seq_err, hist, head,
                      count, sl_max, n_short=10, n_long=30, delta=0.85, eps=1e-6, sl_min=2.0, sl_hi=None, pad_id=-1,
                      row_lse=None, draft_entropy=False, budget=None, out=None, stream=None):
    """``dsde_shard_accept_step``: call 2 with the signal update and the SL rule
    fused behind it (hist/head/count updated in place).  Returns the outputs of
    shard_accept plus mu_last, var_short, var_long, wvir, sf, sl_hat, sl_cap,
    sl_next."""
    lib = load()
    out, args, _keep = _shard_accept_call(parts, V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max,
                                          seq_err, pad_id, row_lse, draft_entropy, out, stream)
    B = int(sl.shape[0])
    W = int(hist.shape[1])
    sl_hi = k_max if sl_hi is None else sl_hi
    dev = sl.device
    f32 = torch.float32
    for k in ("mu_last", "var_short", "var_long", "wvir", "sf", "sl_hat"):
        if k not in out:
            out[k] = torch.empty(B, dtype=f32, device=dev)
    if "sl_cap" not in out:
        out["sl_cap"] = torch.empty(1, dtype=f32, device=dev)
    if "sl_next" not in out:
        out["sl_next"] = torch.empty(B, dtype=torch.int32, device=dev)
    rc = lib.dsde_shard_accept_step(
        *args, _ptr(hist, f32, B * W, "hist"), _ptr(head, torch.int32, B, "head"),
        _ptr(count, torch.int32, B, "count"), W, n_short, n_long, float(delta), float(eps),
        _ptr(out["mu_last"], f32, B), _ptr(out["var_short"], f32, B), _ptr(out["var_long"], f32, B),
        _ptr(out["wvir"], f32, B), _ptr(out["sf"], f32, B), _ptr(sl_max, f32, B, "sl_max"), float(sl_min),
        int(sl_hi), _ptr(budget, torch.int32, B, "budget") if budget is not None else None,
        _ptr(out["sl_hat"], f32, B), _ptr(out["sl_cap"], f32, 1), _ptr(out["sl_next"], torch.int32, B),
        _ptr(seq_err, None, B, "seq_err"), _stream(stream))
    _check(rc)
    return out


def shard_draw_mass(target, draft, v_begin, part, jobs, k_max, workspace, mass=None, stream=None):
    """``dsde_shard_draw_mass`` (call 3).  Returns mass [B, 32] uint8 records."""
    lib = load()
    B = int(jobs.shape[0])
    dt, V_shard, N = _shard_rows(target, draft, B)
    if mass is None:
        mass = torch.empty((B, SHARD_MASS_BYTES), dtype=torch.uint8, device=target.device)
    rc = lib.dsde_shard_draw_mass(
        _ptr(target, name="target"), _ptr(draft, name="draft") if N > 0 else None, dt, V_shard, int(v_begin), B, N,
        k_max, _ptr(part, torch.uint8, N * SHARD_PARTIAL_BYTES, "part") if N > 0 else None,
        _ptr(jobs, torch.uint8, B * DRAW_JOB_BYTES, "jobs"), _ptr(mass, torch.uint8, B * SHARD_MASS_BYTES, "mass"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(), _stream(stream))
    _check(rc)
    return mass


def shard_draw_pick(g, masses, target, draft, v_begin, jobs, k_max, accepted, tokens, seq_err, workspace,
                    pad_id=-1, drawn=None, stream=None):
    """``dsde_shard_draw_pick`` (call 4) for shard g from the gathered masses
    [G, B, 32] (uint8, shard order).  accepted, tokens and seq_err are updated in
    place; returns drawn [B] int32 (the token where this shard determined it,
    else -1)."""
    lib = load()
    G = int(masses.shape[0])
    B = int(jobs.shape[0])
    dt, V_shard, N = _shard_rows(target, draft, B)
    if drawn is None:
        drawn = torch.empty(B, dtype=torch.int32, device=target.device)
    rc = lib.dsde_shard_draw_pick(
        G, int(g), _ptr(masses, torch.uint8, G * B * SHARD_MASS_BYTES, "masses"), _ptr(target, name="target"),
        _ptr(draft, name="draft") if N > 0 else None, dt, V_shard, int(v_begin), B, N, k_max,
        _ptr(jobs, torch.uint8, B * DRAW_JOB_BYTES, "jobs"), int(pad_id),
        _ptr(accepted, torch.int32, B, "accepted"), _ptr(tokens, torch.int32, B * (k_max + 1), "tokens"),
        _ptr(drawn, torch.int32, B, "drawn"), _ptr(seq_err, None, B, "seq_err"),
        _ptr(workspace, torch.uint8, None, "workspace"), workspace.numel(), _stream(stream))
    _check(rc)
    return drawn


def slice_bounds(V, G):
    """Boundaries of G near-equal contiguous vocabulary slices (multiples of 8
    where the width allows, so that bf16 slices keep 16-byte rows)."""
    step = -(-V // G)
    step = -(-step // 8) * 8 if step * (G - 1) < V else step
    bounds = [min(g * step, V) for g in range(G)] + [V]
    return [(bounds[g], bounds[g + 1]) for g in range(G) if bounds[g + 1] > bounds[g]]


def verify_sharded(target, draft, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, slices,
                   pad_id=-1, row_lse=None, draft_entropy=False):
    """The four shard calls for every slice of ``slices`` ([(v_begin, v_end), ...],
    ascending, tiling [0, V)) run on one device, the exchanges being the gathered
    tensors themselves: the sharded path's results on one GPU, for tests and
    measurements.  Returns the dict of dsde_verify's outputs plus ``drawn``
    (the all-reduce max of every shard's drawn[]) and the two exchanged arrays,
    ``parts`` [G, N, 64] and ``masses`` [G, B, 32]."""
    V = int(target.shape[1])
    B = int(sl.shape[0])
    N = int(draft.shape[0]) if draft is not None else 0
    dev = target.device
    shards = []
    for (v0, v1) in slices:
        t = target[:, v0:v1].contiguous()
        d = draft[:, v0:v1].contiguous() if N > 0 else None
        ws = new_shard_workspace(B, N, v1 - v0, k_max, device=dev)
        shards.append((v0, t, d, ws))
    parts, errs = [], []
    for (v0, t, d, ws) in shards:
        p, e = shard_stats(t, d, v0, V, sl, cu_sl, draft_tokens, temperature, k_max, ws)
        parts.append(p[:max(N, 1)])
        errs.append(e)
    seq_err = errs[0].clone()
    out = shard_accept(torch.stack(parts), V, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, k_max, seq_err,
                       pad_id=pad_id, row_lse=row_lse, draft_entropy=draft_entropy)
    masses = torch.stack([shard_draw_mass(t, d, v0, p, out["jobs"], k_max, ws)
                          for (v0, t, d, ws), p in zip(shards, parts)])
    drawn = [shard_draw_pick(g, masses, t, d, v0, out["jobs"], k_max, out["accepted"], out["tokens"], seq_err, ws,
                             pad_id=pad_id)
             for g, (v0, t, d, ws) in enumerate(shards)]
    out["drawn"] = torch.stack(drawn).max(dim=0).values
    out["shard_seq_err"] = errs
    out["parts"] = torch.stack(parts)
    out["masses"] = masses
    return out

