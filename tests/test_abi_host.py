"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function include/dsde.h declares, and
reject invalid arguments before any HIP call (fake non-null host pointers are
used, which the library never dereferences on these paths).
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dsde.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2509_01083_amd as dsde
    if not os.path.exists(dsde.LIB_PATH):
        from paper_2509_01083_amd import build_lib
        build_lib.build()
    return dsde.load()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int32_t|size_t|const char \*)\s*(dsde_\w+)\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("dsde_verify", "dsde_kld_signal", "dsde_next_sl", "dsde_verify_workspace_bytes"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    import paper_2509_01083_amd as dsde
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} is declared but not exported"
    assert sorted(dsde.EXPORTS) == declared_functions()


def test_version_and_status_strings(lib):
    assert lib.dsde_abi_version() == 3
    for code, text in ((0, b"ok"), (1, b"invalid argument"), (2, b"workspace too small"), (3, b"device error")):
        assert lib.dsde_status_string(code) == text
    assert lib.dsde_status_string(99) == b"unknown status"


def test_workspace_sizes(lib):
    ws = lib.dsde_verify_workspace_bytes
    assert ws(256, 1152, 128256, 8) > 0
    assert ws(256, 1152, 128256, 8) >= ws(256, 100, 128256, 8)
    assert ws(4, 8, 4194304, 4) > 0  # the largest vocabulary (DSDE_MAX_VOCAB)
    for bad in ((0, 0, 10, 4), (4, -1, 10, 4), (4, 0, 0, 4), (4, 0, 4194305, 4), (4, 0, 1 << 31, 4),
                (4, 0, 10, -1), (4, 0, 10, 64), (4, 17, 10, 4)):
        assert ws(*bad) == 0, bad


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def verify_args(**over):
    a = dict(target=FAKE, draft=FAKE, dtype=1, V=1000, B=4, N=8, k_max=4, sl=FAKE, cu_sl=FAKE, toks=FAKE,
             temp=FAKE, u_acc=FAKE, u_res=FAKE, pad=-1, acc=FAKE, tokens=FAKE, kld=FAKE, err=FAKE, lse=None,
             ent=None, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(over)
    return list(a.values())


@pytest.mark.parametrize("over", [
    dict(dtype=2), dict(dtype=-1), dict(V=0), dict(V=4194305), dict(V=1 << 31), dict(B=0), dict(N=-1), dict(k_max=-1),
    dict(k_max=64), dict(N=17), dict(target=None), dict(sl=None), dict(cu_sl=None), dict(temp=None),
    dict(u_res=None), dict(acc=None), dict(tokens=None), dict(err=None), dict(ws=None), dict(draft=None),
    dict(toks=None), dict(u_acc=None), dict(kld=None), dict(ws=ctypes.c_void_p(0x1001)),
])
def test_verify_rejects_invalid_arguments(lib, over):
    assert lib.dsde_verify(*verify_args(**over)) == 1


def test_verify_allows_missing_draft_arrays_when_nothing_is_drafted(lib):
    # N = 0: draft arrays may be NULL; with a tiny workspace the next check fires instead
    rc = lib.dsde_verify(*verify_args(N=0, draft=None, toks=None, u_acc=None, kld=None, ws_bytes=16))
    assert rc == 2


def test_verify_workspace_too_small(lib):
    need = lib.dsde_verify_workspace_bytes(4, 8, 1000, 4)
    assert lib.dsde_verify(*verify_args(ws_bytes=need - 1)) == 2


def signal_args(**over):
    a = dict(B=4, N=8, sl=FAKE, cu=FAKE, kld=FAKE, hist=FAKE, head=FAKE, count=FAKE, W=32, ns=10, nl=30,
             delta=0.85, eps=1e-6, mu=FAKE, vs=FAKE, vl=FAKE, wvir=FAKE, sf=FAKE, err=FAKE, stream=None)
    a.update(over)
    return list(a.values())


@pytest.mark.parametrize("over", [
    dict(B=0), dict(N=-1), dict(W=0), dict(ns=0), dict(ns=31), dict(delta=0.0), dict(delta=1.5),
    dict(delta=float("nan")), dict(eps=-1.0), dict(eps=0.0), dict(eps=float("inf")), dict(sl=None), dict(hist=None),
    dict(head=None), dict(count=None), dict(mu=None), dict(sf=None), dict(err=None), dict(kld=None),
])
def test_kld_signal_rejects_invalid_arguments(lib, over):
    assert lib.dsde_kld_signal(*signal_args(**over)) == 1


@pytest.mark.parametrize("over", [
    dict(B=0), dict(sl_min=float("nan")), dict(sl_min=9.0), dict(sl_min=8.5), dict(sf=None), dict(wvir=None),
    dict(sl_max=None), dict(hat=None), dict(cap=None), dict(nxt=None), dict(err=None),
])
def test_next_sl_rejects_invalid_arguments(lib, over):
    a = dict(B=4, sf=FAKE, wvir=FAKE, sl_max=FAKE, sl_min=2.0, sl_hi=8, budget=None, hat=FAKE, cap=FAKE, nxt=FAKE,
             err=FAKE, stream=None)
    a.update(over)
    assert lib.dsde_next_sl(*a.values()) == 1


def test_profile_hook_needs_both_events(lib):
    assert lib.dsde_set_profile_events(FAKE, None) == 1
    assert lib.dsde_set_profile_events(None, None) == 0


def test_binding_never_touches_the_oracle():
    src = open(os.path.join(ROOT, "paper_2509_01083_amd", "__init__.py")).read()
    for f in os.listdir(os.path.join(ROOT, "paper_2509_01083_amd", "csrc")):
        src += open(os.path.join(ROOT, "paper_2509_01083_amd", "csrc", f)).read()
    assert "oracle" not in src.lower()


def test_stream_read_rejects_invalid_arguments(lib):
    fn = lib.dsde_stream_read
    fn.restype = ctypes.c_int32
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    ok_buf, out = ctypes.c_void_p(0x1000), ctypes.c_void_p(0x2000)
    for buf, nbytes, o in ((None, 16, out), (ok_buf, 16, None), (ok_buf, 0, out), (ok_buf, -16, out),
                           (ok_buf, 24, out), (ctypes.c_void_p(0x1008), 16, out)):
        assert fn(buf, nbytes, o, None) == 1


@pytest.mark.parametrize("over", [
    dict(B=0), dict(N=-1), dict(sl=None), dict(cu=None), dict(acc=None), dict(err=None), dict(amax=None),
    dict(ksum=None), dict(kcnt=None), dict(kmax=None), dict(kld=None),
])
def test_calibration_update_rejects_invalid_arguments(lib, over):
    a = dict(B=4, N=8, sl=FAKE, cu=FAKE, acc=FAKE, kld=FAKE, err=FAKE, amax=FAKE, ksum=FAKE, kcnt=FAKE, kmax=FAKE,
             stream=None)
    a.update(over)
    assert lib.dsde_calibration_update(*a.values()) == 1


@pytest.mark.parametrize("over", [
    dict(B=0), dict(eps=-1e-6), dict(eps=float("nan")), dict(pooled=2), dict(amax=None), dict(ksum=None),
    dict(kcnt=None), dict(kmax=None), dict(out=None),
])
def test_calibrate_sl_max_rejects_invalid_arguments(lib, over):
    a = dict(B=4, amax=FAKE, ksum=FAKE, kcnt=FAKE, kmax=FAKE, eps=1e-6, pooled=0, out=FAKE, stream=None)
    a.update(over)
    assert lib.dsde_calibrate_sl_max(*a.values()) == 1


def test_shard_workspace_sizes(lib):
    ws = lib.dsde_shard_workspace_bytes
    assert ws(256, 1152, 16032, 8) > 0
    assert ws(256, 1152, 16032, 8) > lib.dsde_verify_workspace_bytes(256, 1152, 16032, 8)
    for bad in ((0, 0, 10, 4), (4, 0, 0, 4), (4, 0, 4194305, 4), (4, 17, 10, 4), (4, 0, 10, 64)):
        assert ws(*bad) == 0, bad


def shard_stats_args(**over):
    a = dict(target=FAKE, draft=FAKE, dtype=1, V_shard=500, v_begin=500, V=1000, B=4, N=8, k_max=4, sl=FAKE,
             cu_sl=FAKE, toks=FAKE, temp=FAKE, part=FAKE, err=FAKE, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(over)
    return list(a.values())


@pytest.mark.parametrize("over", [
    dict(dtype=2), dict(V_shard=0), dict(v_begin=-1), dict(v_begin=501), dict(V=4194305), dict(V=0), dict(B=0),
    dict(N=17), dict(k_max=64), dict(target=None), dict(draft=None), dict(sl=None), dict(cu_sl=None),
    dict(toks=None), dict(temp=None), dict(part=None), dict(err=None), dict(ws=None),
    dict(ws=ctypes.c_void_p(0x1001)),
])
def test_shard_stats_rejects_invalid_arguments(lib, over):
    assert lib.dsde_shard_stats(*shard_stats_args(**over)) == 1


def test_shard_stats_workspace_too_small(lib):
    need = lib.dsde_shard_workspace_bytes(4, 8, 500, 4)
    assert lib.dsde_shard_stats(*shard_stats_args(ws_bytes=need - 1)) == 2


@pytest.mark.parametrize("over", [
    dict(G=0), dict(G=1025), dict(V=0), dict(B=0), dict(N=17), dict(parts=None), dict(sl=None), dict(toks=None),
    dict(u_acc=None), dict(u_res=None), dict(acc=None), dict(tokens=None), dict(kld=None), dict(jobs=None),
    dict(err=None),
])
def test_shard_accept_rejects_invalid_arguments(lib, over):
    a = dict(G=2, parts=FAKE, V=1000, B=4, N=8, k_max=4, sl=FAKE, cu_sl=FAKE, toks=FAKE, temp=FAKE, u_acc=FAKE,
             u_res=FAKE, pad=-1, acc=FAKE, tokens=FAKE, kld=FAKE, lse=None, ent=None, jobs=FAKE, err=FAKE,
             stream=None)
    a.update(over)
    assert lib.dsde_shard_accept(*a.values()) == 1


@pytest.mark.parametrize("over", [
    dict(G=0), dict(B=0), dict(parts=None), dict(jobs=None), dict(err=None), dict(W=0), dict(n_short=0),
    dict(n_short=31), dict(delta=0.0), dict(delta=1.5), dict(eps=-1.0), dict(eps=0.0), dict(hist=None), dict(sf=None),
    dict(sl_max=None), dict(sl_min=float("nan")), dict(sl_min=9.0), dict(sl_next=None),
])
def test_shard_accept_step_rejects_invalid_arguments(lib, over):
    """The fused call 2 checks call 2's arguments and the signal and SL-rule
    arguments of dsde_step before anything is enqueued."""
    a = dict(G=2, parts=FAKE, V=1000, B=4, N=8, k_max=4, sl=FAKE, cu_sl=FAKE, toks=FAKE, temp=FAKE, u_acc=FAKE,
             u_res=FAKE, pad=-1, acc=FAKE, tokens=FAKE, kld=FAKE, lse=None, ent=None, jobs=FAKE,
             hist=FAKE, head=FAKE, count=FAKE, W=32, n_short=10, n_long=30, delta=0.85, eps=1e-6,
             mu_last=FAKE, var_short=FAKE, var_long=FAKE, wvir=FAKE, sf=FAKE, sl_max=FAKE, sl_min=2.0, sl_hi=8,
             budget=None, sl_hat=FAKE, sl_cap=FAKE, sl_next=FAKE, err=FAKE, stream=None)
    a.update(over)
    assert lib.dsde_shard_accept_step(*a.values()) == 1


@pytest.mark.parametrize("over", [
    dict(dtype=2), dict(V_shard=0), dict(v_begin=-1), dict(B=0), dict(target=None), dict(draft=None),
    dict(part=None), dict(jobs=None), dict(mass=None), dict(ws=None),
])
def test_shard_draw_mass_rejects_invalid_arguments(lib, over):
    a = dict(target=FAKE, draft=FAKE, dtype=1, V_shard=500, v_begin=0, B=4, N=8, k_max=4, part=FAKE, jobs=FAKE,
             mass=FAKE, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(over)
    assert lib.dsde_shard_draw_mass(*a.values()) == 1


@pytest.mark.parametrize("over", [
    dict(G=0), dict(g=-1), dict(g=2), dict(G=1025), dict(masses=None), dict(target=None), dict(draft=None),
    dict(dtype=2), dict(jobs=None), dict(acc=None), dict(tokens=None), dict(drawn=None), dict(err=None),
    dict(ws=None),
])
def test_shard_draw_pick_rejects_invalid_arguments(lib, over):
    a = dict(G=2, g=1, masses=FAKE, target=FAKE, draft=FAKE, dtype=1, V_shard=500, v_begin=500, B=4, N=8,
             k_max=4, jobs=FAKE, pad=-1, acc=FAKE, tokens=FAKE, drawn=FAKE, err=FAKE, ws=FAKE, ws_bytes=1 << 30,
             stream=None)
    a.update(over)
    assert lib.dsde_shard_draw_pick(*a.values()) == 1


def test_slice_bounds_tile_the_vocabulary():
    import paper_2509_01083_amd as dsde
    for V, G in ((128256, 8), (25281, 3), (17, 4), (100, 8), (1, 3), (152064, 7)):
        b = dsde.slice_bounds(V, G)
        assert b[0][0] == 0 and b[-1][1] == V and len(b) <= G
        assert all(b[i][1] == b[i + 1][0] and b[i][0] < b[i][1] for i in range(len(b) - 1))


def _step_static_args(**over):
    a = dict(target=FAKE, draft=FAKE, dtype=1, V=1000, B=4, N=8, k_max=4, sl=FAKE, cu_sl=FAKE, toks=FAKE,
             temp=FAKE, u_acc=FAKE, u_res=FAKE, pad=-1, acc=FAKE, tokens=FAKE, kld=FAKE, lse=None, ent=None,
             hist=FAKE, head=FAKE, count=FAKE, W=32, n_short=10, n_long=30, delta=0.85, eps=1e-6,
             mu_last=FAKE, var_short=FAKE, var_long=FAKE, wvir=FAKE, sf=FAKE, sl_max=FAKE, sl_min=2.0, sl_hi=8,
             budget=None, sl_hat=FAKE, sl_cap=FAKE, sl_next=FAKE, err=FAKE, stream=None)
    a.update(over)
    return list(a.values())


@pytest.mark.parametrize("over", [
    dict(dtype=2), dict(B=0), dict(V=0), dict(k_max=64), dict(target=None), dict(draft=None), dict(acc=None),
    dict(err=None), dict(W=0), dict(n_short=31), dict(eps=0.0), dict(hist=None), dict(sl_max=None),
    dict(sl_min=9.0), dict(sl_next=None),
])
def test_step_static_rejects_invalid_arguments(lib, over):
    """The allocation-free fused step checks dsde_step's arguments (less the
    workspace) before any HIP call."""
    assert lib.dsde_step_static(*_step_static_args(**over)) == 1


def test_step_static_rejects_shapes_beyond_its_scratch(lib):
    import paper_2509_01083_amd as dsde
    # B = 1024 sequences with k_max = 63 at V = 128256 need ~56 MB of scratch
    B, k_max, V = 1024, 63, 128256
    N = B * k_max
    assert lib.dsde_verify_workspace_bytes(B, N, V, k_max) > dsde.STATIC_SCRATCH_BYTES
    assert lib.dsde_step_static(*_step_static_args(B=B, N=N, V=V, k_max=k_max, sl_hi=63)) == 2
    # every configuration of the benchmark fits
    for B, N, V, k in ((256, 2048, 128256, 8), (512, 8192, 152064, 16), (1024, 8192, 128256, 8)):
        assert 0 < lib.dsde_verify_workspace_bytes(B, N, V, k) <= dsde.STATIC_SCRATCH_BYTES


def test_static_scratch_size_matches_header():
    import paper_2509_01083_amd as dsde
    m = re.search(r"#define DSDE_STATIC_SCRATCH_BYTES \((\d+)u << (\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == dsde.STATIC_SCRATCH_BYTES
