"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any HIP call
(so no call here reaches the runtime; fake device addresses are never used)."""
import ctypes
import os
import re

import pytest

from paper_2609_36757_amd import fastvr

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "fastvr.h")

# Distinct fake addresses, 1 TiB apart, for calls that must fail validation:
# every case below is rejected on the host before the HIP runtime is touched.
Q, K, V, O, LSE, RK, RV, DO, DQ, DK, DV, RS, Z, VEL, ZH, X, TL, OUT = ((i + 1) << 40 for i in range(18))
BIG = 1 << 62


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fastvr_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fastvr.LIB_PATH):
        pytest.fail("libfastvr.so is not built (run `python -m paper_2609_36757_amd.build`)")
    return fastvr.load()


def test_header_symbols_exported(lib):
    declared = _declared_functions()
    assert set(declared) == set(fastvr.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_version_and_status_strings(lib):
    assert lib.fastvr_abi_version() == 7
    assert lib.fastvr_status_string(0) == b"FASTVR_OK"
    assert lib.fastvr_status_string(1) == b"FASTVR_ERR_INVALID_ARGUMENT"
    assert lib.fastvr_status_string(2) == b"FASTVR_ERR_UNSUPPORTED"
    assert lib.fastvr_status_string(3) == b"FASTVR_ERR_CAPACITY"
    assert lib.fastvr_status_string(4) == b"FASTVR_ERR_HIP"
    assert lib.fastvr_status_string(99) == b"FASTVR_ERR_UNKNOWN"


GOOD = dict(q=Q, k=K, v=V, o=O, lse=LSE, B=1, H=2, Nq=64, Nkv=64, d=64, chunk_len=16, q_chunk_offset=0,
            window_chunks=-1, scale=0.125)


def _fwd(**kw):
    a = dict(GOOD)
    a.update(kw)
    return fastvr.fwd_raw(a["q"], a["k"], a["v"], a["o"], a["lse"], a["B"], a["H"], a["Nq"], a["Nkv"], a["d"],
                          a["chunk_len"], a["q_chunk_offset"], a["window_chunks"], a["scale"], None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(q=None), fastvr.ERR_INVALID_ARGUMENT, "q is NULL"),
    (dict(k=None), fastvr.ERR_INVALID_ARGUMENT, "k is NULL"),
    (dict(v=None), fastvr.ERR_INVALID_ARGUMENT, "v is NULL"),
    (dict(o=None), fastvr.ERR_INVALID_ARGUMENT, "o is NULL"),
    (dict(q=Q + 8), fastvr.ERR_INVALID_ARGUMENT, "aligned"),
    (dict(o=O + 4), fastvr.ERR_INVALID_ARGUMENT, "aligned"),
    (dict(lse=LSE + 2), fastvr.ERR_INVALID_ARGUMENT, "lse is not 4-byte aligned"),
    (dict(B=-1), fastvr.ERR_INVALID_ARGUMENT, "negative size"),
    (dict(Nkv=-5), fastvr.ERR_INVALID_ARGUMENT, "negative size"),
    (dict(d=96), fastvr.ERR_UNSUPPORTED, "head_dim"),
    (dict(d=256), fastvr.ERR_UNSUPPORTED, "head_dim"),
    (dict(chunk_len=0), fastvr.ERR_INVALID_ARGUMENT, "chunk_len"),
    (dict(q_chunk_offset=-1), fastvr.ERR_INVALID_ARGUMENT, "q_chunk_offset"),
    (dict(window_chunks=-2), fastvr.ERR_INVALID_ARGUMENT, "window_chunks"),
    (dict(scale=float("nan")), fastvr.ERR_INVALID_ARGUMENT, "scale"),
    (dict(scale=float("inf")), fastvr.ERR_INVALID_ARGUMENT, "scale"),
    (dict(Nkv=63), fastvr.ERR_INVALID_ARGUMENT, "would not see its own key"),
    (dict(Nq=16, q_chunk_offset=4), fastvr.ERR_INVALID_ARGUMENT, "would not see its own key"),
    (dict(q_chunk_offset=BIG, chunk_len=16), fastvr.ERR_INVALID_ARGUMENT, "overflows"),
    (dict(Nq=BIG, Nkv=BIG), fastvr.ERR_INVALID_ARGUMENT, "overflows"),
    (dict(Nq=1 << 31, Nkv=1 << 31), fastvr.ERR_UNSUPPORTED, "2^31"),
    (dict(o=Q + 64), fastvr.ERR_INVALID_ARGUMENT, "overlaps"),
    (dict(lse=O + 16), fastvr.ERR_INVALID_ARGUMENT, "overlaps"),
])
def test_fwd_rejects(lib, kw, status, needle):
    assert _fwd(**kw) == status
    assert needle in fastvr.last_error()


def test_fwd_too_many_workgroups(lib):
    # chunk_len 1 -> one 256-row tile per query row: B*H*Nq = 2^23 items exceed one launch
    assert _fwd(B=1, H=64, Nq=1 << 17, Nkv=1 << 17, chunk_len=1) == fastvr.ERR_UNSUPPORTED
    assert "workgroups" in fastvr.last_error()


@pytest.mark.parametrize("kw", [dict(Nq=0), dict(B=0), dict(H=0), dict(Nq=0, q=None, o=None)])
def test_fwd_empty_problem_is_ok(lib, kw):
    assert _fwd(**kw) == fastvr.OK
    assert fastvr.last_error() == ""


def _fwd_ex(**kw):
    a = dict(GOOD, B=2, q_sb=64 * 128, q_st=128, k_sb=64 * 128, k_st=128, v_sb=64 * 128, v_st=128,
             o_sb=64 * 128, o_st=128, o_bf16=0)
    a.update(kw)
    return fastvr.fwd_ex_raw(a["q"], a["q_sb"], a["q_st"], a["k"], a["k_sb"], a["k_st"], a["v"], a["v_sb"],
                             a["v_st"], a["o"], a["o_sb"], a["o_st"], a["o_bf16"], a["lse"], a["B"], a["H"],
                             a["Nq"], a["Nkv"], a["d"], a["chunk_len"], a["q_chunk_offset"], a["window_chunks"],
                             a["scale"], None)


@pytest.mark.parametrize("kw,needle", [
    (dict(q_st=64), "token stride"),
    (dict(k_st=132), "multiples of 8"),
    (dict(o_st=130), "multiples of 4"),
    (dict(v_sb=100 * 128 + 4), "multiples of 8"),
    (dict(o_sb=63 * 128), "batch stride"),
    (dict(k_sb=BIG, k_st=BIG // 4), "overflows"),
    (dict(o_bf16=2), "o_bf16 must be 0 or 1"),
    (dict(o_bf16=1, o_st=132), "multiples of 8"),       # bf16 O rows: 16-byte strides are multiples of 8
    (dict(o_bf16=1, o=O + 8), "aligned"),
])
def test_fwd_ex_rejects_bad_strides(lib, kw, needle):
    assert _fwd_ex(**kw) == fastvr.ERR_INVALID_ARGUMENT
    assert needle in fastvr.last_error()


def _app(**kw):
    a = dict(kc=Q, vc=K, kn=V, vn=O, B=1, H=2, d=64, capacity=100, cache_len=10, n_new=20)
    a.update(kw)
    return fastvr.append_raw(a["kc"], a["vc"], a["kn"], a["vn"], a["B"], a["H"], a["d"], a["capacity"],
                             a["cache_len"], a["n_new"], None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(capacity=29), fastvr.ERR_CAPACITY, "capacity"),
    (dict(cache_len=81), fastvr.ERR_CAPACITY, "capacity"),
    (dict(kc=None), fastvr.ERR_INVALID_ARGUMENT, "k_cache is NULL"),
    (dict(vn=None), fastvr.ERR_INVALID_ARGUMENT, "v_new is NULL"),
    (dict(kn=V + 2), fastvr.ERR_INVALID_ARGUMENT, "aligned"),
    (dict(d=32), fastvr.ERR_UNSUPPORTED, "head_dim"),
    (dict(n_new=-1), fastvr.ERR_INVALID_ARGUMENT, "negative"),
    (dict(cache_len=BIG, n_new=BIG, capacity=BIG), fastvr.ERR_INVALID_ARGUMENT, "overflows"),
    (dict(vc=Q + 256), fastvr.ERR_INVALID_ARGUMENT, "overlap"),
    (dict(kn=Q + 1024), fastvr.ERR_INVALID_ARGUMENT, "overlaps"),
    (dict(B=70000, capacity=30), fastvr.ERR_UNSUPPORTED, "65535"),
])
def test_append_rejects(lib, kw, status, needle):
    assert _app(**kw) == status
    assert needle in fastvr.last_error()


@pytest.mark.parametrize("kw", [dict(n_new=0), dict(B=0), dict(H=0)])
def test_append_empty_is_ok(lib, kw):
    assert _app(**kw) == fastvr.OK


RING_GOOD = dict(q=Q, k=K, v=V, rk=RK, rv=RV, o=O, lse=LSE, B=1, H=2, n_new=64, d=128, chunk_len=64,
                 chunk_index=3, window_chunks=1, scale=0.125)


def _ring(**kw):
    a = dict(RING_GOOD)
    a.update(kw)
    return fastvr.ring_step_raw(a["q"], a["k"], a["v"], a["rk"], a["rv"], a["o"], a["lse"], a["B"], a["H"],
                                a["n_new"], a["d"], a["chunk_len"], a["chunk_index"], a["window_chunks"],
                                a["scale"], None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(window_chunks=-1), fastvr.ERR_INVALID_ARGUMENT, "window_chunks >= 0"),
    (dict(window_chunks=8), fastvr.ERR_UNSUPPORTED, "window_chunks 8 > 7"),
    (dict(n_new=0), fastvr.ERR_INVALID_ARGUMENT, "n_new"),
    (dict(n_new=65), fastvr.ERR_INVALID_ARGUMENT, "n_new"),
    (dict(chunk_len=66, n_new=60), fastvr.ERR_UNSUPPORTED, "multiple of 4"),
    (dict(chunk_len=68, n_new=60, d=64), fastvr.ERR_UNSUPPORTED, "multiple of 8"),
    (dict(chunk_index=-1), fastvr.ERR_INVALID_ARGUMENT, "chunk_index"),
    (dict(d=96), fastvr.ERR_UNSUPPORTED, "head_dim"),
    (dict(rk=None), fastvr.ERR_INVALID_ARGUMENT, "k_ring or v_ring is NULL"),
    (dict(rv=RV + 8), fastvr.ERR_INVALID_ARGUMENT, "16-byte aligned"),
    (dict(q=None), fastvr.ERR_INVALID_ARGUMENT, "q is NULL"),
    (dict(scale=float("nan")), fastvr.ERR_INVALID_ARGUMENT, "scale"),
    (dict(rk=O + 256), fastvr.ERR_INVALID_ARGUMENT, "ring overlaps"),
    (dict(rk=K + 512), fastvr.ERR_INVALID_ARGUMENT, "ring overlaps"),
    (dict(rv=RK + 4096), fastvr.ERR_INVALID_ARGUMENT, "k_ring and v_ring overlap"),
    (dict(B=-1), fastvr.ERR_INVALID_ARGUMENT, "negative size"),
    (dict(chunk_len=1 << 40, n_new=64), fastvr.ERR_UNSUPPORTED, "2^31"),
])
def test_ring_step_rejects(lib, kw, status, needle):
    assert _ring(**kw) == status
    assert needle in fastvr.last_error()


@pytest.mark.parametrize("kw", [dict(B=0), dict(H=0)])
def test_ring_step_empty_is_ok(lib, kw):
    assert _ring(**kw) == fastvr.OK


BWD_GOOD = dict(q=Q, k=K, v=V, o=O, lse=LSE, dout=DO, dq=DQ, dk=DK, dv=DV, rs=RS, B=1, H=2, Nq=64, Nkv=64, d=64,
                chunk_len=16, q_chunk_offset=0, window_chunks=-1, scale=0.125)


def _bwd(**kw):
    a = dict(BWD_GOOD)
    a.update(kw)
    return fastvr.bwd_raw(a["q"], a["k"], a["v"], a["o"], a["lse"], a["dout"], a["dq"], a["dk"], a["dv"], a["rs"],
                          a["B"], a["H"], a["Nq"], a["Nkv"], a["d"], a["chunk_len"], a["q_chunk_offset"],
                          a["window_chunks"], a["scale"], None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(q=None), fastvr.ERR_INVALID_ARGUMENT, "q is NULL"),
    (dict(dout=None), fastvr.ERR_INVALID_ARGUMENT, "dout is NULL"),
    (dict(o=None), fastvr.ERR_INVALID_ARGUMENT, "o is NULL"),
    (dict(dq=None), fastvr.ERR_INVALID_ARGUMENT, "dq is NULL"),
    (dict(dk=None), fastvr.ERR_INVALID_ARGUMENT, "dk is NULL"),
    (dict(dv=None), fastvr.ERR_INVALID_ARGUMENT, "dv is NULL"),
    (dict(lse=None), fastvr.ERR_INVALID_ARGUMENT, "lse or row_stats is NULL"),
    (dict(rs=None), fastvr.ERR_INVALID_ARGUMENT, "lse or row_stats is NULL"),
    (dict(dk=DK + 8), fastvr.ERR_INVALID_ARGUMENT, "aligned"),
    (dict(rs=RS + 2), fastvr.ERR_INVALID_ARGUMENT, "4-byte aligned"),
    (dict(B=-1), fastvr.ERR_INVALID_ARGUMENT, "negative size"),
    (dict(d=96), fastvr.ERR_UNSUPPORTED, "head_dim"),
    (dict(chunk_len=0), fastvr.ERR_INVALID_ARGUMENT, "chunk_len"),
    (dict(q_chunk_offset=-1), fastvr.ERR_INVALID_ARGUMENT, "q_chunk_offset"),
    (dict(window_chunks=-2), fastvr.ERR_INVALID_ARGUMENT, "window_chunks"),
    (dict(scale=float("nan")), fastvr.ERR_INVALID_ARGUMENT, "scale"),
    (dict(Nkv=63), fastvr.ERR_INVALID_ARGUMENT, "would not see its own key"),
    (dict(Nkv=0), fastvr.ERR_INVALID_ARGUMENT, "no keys"),
    (dict(Nkv=1 << 31, Nq=64), fastvr.ERR_UNSUPPORTED, "2^31"),
    (dict(H=1 << 16), fastvr.ERR_UNSUPPORTED, "H * d"),
    (dict(dq=Q + 64), fastvr.ERR_INVALID_ARGUMENT, "dq overlaps q"),
    (dict(dk=DV), fastvr.ERR_INVALID_ARGUMENT, "dk overlaps dv"),
    (dict(rs=LSE), fastvr.ERR_INVALID_ARGUMENT, "row_stats overlaps lse"),
    (dict(dv=K + 4096), fastvr.ERR_INVALID_ARGUMENT, "dv overlaps k"),
])
def test_bwd_rejects(lib, kw, status, needle):
    assert _bwd(**kw) == status
    assert needle in fastvr.last_error()


@pytest.mark.parametrize("kw", [dict(B=0), dict(H=0), dict(Nq=0, Nkv=0)])
def test_bwd_empty_is_ok(lib, kw):
    assert _bwd(**kw) == fastvr.OK


def _bwd_na(**kw):
    a = dict(BWD_GOOD)
    a.update(kw)
    return fastvr.bwd_noalloc_raw(a["q"], a["k"], a["v"], a["o"], a["lse"], a["dout"], a["dq"], a["dk"], a["dv"],
                                  a["B"], a["H"], a["Nq"], a["Nkv"], a["d"], a["chunk_len"], a["q_chunk_offset"],
                                  a["window_chunks"], a["scale"], None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(q=None), fastvr.ERR_INVALID_ARGUMENT, "q is NULL"),
    (dict(lse=None), fastvr.ERR_INVALID_ARGUMENT, "lse is NULL"),
    (dict(lse=LSE + 2), fastvr.ERR_INVALID_ARGUMENT, "lse is not 4-byte aligned"),
    (dict(dk=DK + 8), fastvr.ERR_INVALID_ARGUMENT, "aligned"),
    (dict(d=96), fastvr.ERR_UNSUPPORTED, "head_dim"),
    (dict(Nkv=63), fastvr.ERR_INVALID_ARGUMENT, "would not see its own key"),
    (dict(dq=Q + 64), fastvr.ERR_INVALID_ARGUMENT, "dq overlaps q"),
    (dict(dv=LSE), fastvr.ERR_INVALID_ARGUMENT, "dv overlaps lse"),
    # 2 * B * H * Nq above the 8 Mi floats of the static workspace
    (dict(H=64, Nq=65537, Nkv=65537), fastvr.ERR_UNSUPPORTED, "at most 8388608"),
])
def test_bwd_noalloc_rejects(lib, kw, status, needle):
    assert _bwd_na(**kw) == status
    assert needle in fastvr.last_error()


@pytest.mark.parametrize("kw", [dict(B=0), dict(H=0), dict(Nq=0, Nkv=0)])
def test_bwd_noalloc_empty_is_ok(lib, kw):
    assert _bwd_na(**kw) == fastvr.OK


OS_GOOD = dict(z=Z, v=VEL, out=ZH, n=1000, sigma=0.5, out_bf16=0)


def _os(**kw):
    a = dict(OS_GOOD)
    a.update(kw)
    return fastvr.one_step_raw(a["z"], a["v"], a["out"], a["n"], a["sigma"], a["out_bf16"], None)


@pytest.mark.parametrize("kw,needle", [
    (dict(z=None), "z_lq is NULL"),
    (dict(v=None), "v is NULL"),
    (dict(out=None), "z_hat is NULL"),
    (dict(z=Z + 8), "aligned"),
    (dict(out=ZH + 4), "aligned"),
    (dict(n=-1), "negative size"),
    (dict(sigma=float("nan")), "sigma"),
    (dict(sigma=float("-inf")), "sigma"),
    (dict(out_bf16=2), "out_bf16"),
    (dict(out=Z), "z_hat overlaps z_lq"),               # fp32 output onto the bf16 input
    (dict(out=Z + 1024, out_bf16=1), "z_hat overlaps z_lq"),
    (dict(out=VEL + 16, out_bf16=1), "z_hat overlaps v"),
])
def test_one_step_rejects(lib, kw, needle):
    assert _os(**kw) == fastvr.ERR_INVALID_ARGUMENT
    assert needle in fastvr.last_error()


def test_one_step_empty_is_ok(lib):
    assert _os(n=0) == fastvr.OK
    assert _os(n=0, z=None, v=None, out=None) == fastvr.OK


TILE_GOOD = dict(x=X, tiles=TL, out=OUT, z=Z, sigma=0.5, B=1, T=2, Hg=68, Wg=120, C=48, tile=64, overlap=16)


def _tg(**kw):
    a = dict(TILE_GOOD)
    a.update(kw)
    return fastvr.tile_gather_raw(a["x"], a["tiles"], a["B"], a["T"], a["Hg"], a["Wg"], a["C"], a["tile"],
                                  a["overlap"], None)


def _tb(update=False, **kw):
    a = dict(TILE_GOOD)
    a.update(kw)
    if update:
        return fastvr.tile_blend_update_raw(a["tiles"], a["z"], a["out"], a["sigma"], a["B"], a["T"], a["Hg"], a["Wg"],
                                            a["C"], a["tile"], a["overlap"], None)
    return fastvr.tile_blend_raw(a["tiles"], a["out"], a["B"], a["T"], a["Hg"], a["Wg"], a["C"], a["tile"],
                                 a["overlap"], None)


def test_tile_axis_host_function(lib):
    assert fastvr.tile_axis(68, 64, 16) == (2, 64)
    assert fastvr.tile_axis(120, 64, 16) == (3, 64)
    assert fastvr.tile_axis(30, 64, 16) == (1, 30)
    with pytest.raises(fastvr.FastVRError):
        fastvr.tile_axis(10, 4, 4)
    with pytest.raises(fastvr.FastVRError):
        fastvr.tile_axis(0, 4, 1)


@pytest.mark.parametrize("fn,kw,status,needle", [
    (_tg, dict(x=None), fastvr.ERR_INVALID_ARGUMENT, "x or tiles is NULL"),
    (_tg, dict(tiles=TL + 8), fastvr.ERR_INVALID_ARGUMENT, "aligned"),
    (_tg, dict(C=44), fastvr.ERR_INVALID_ARGUMENT, "multiple of 8"),
    (_tg, dict(overlap=64), fastvr.ERR_INVALID_ARGUMENT, "overlap < tile"),
    (_tg, dict(overlap=-1), fastvr.ERR_INVALID_ARGUMENT, "overlap < tile"),
    (_tg, dict(tile=5000, overlap=0), fastvr.ERR_UNSUPPORTED, "tile"),
    (_tg, dict(T=-1), fastvr.ERR_INVALID_ARGUMENT, "negative size"),
    (_tg, dict(tiles=X + 1024), fastvr.ERR_INVALID_ARGUMENT, "tiles overlaps x"),
    (_tb, dict(C=46), fastvr.ERR_INVALID_ARGUMENT, "multiple of 4"),
    (_tb, dict(out=None), fastvr.ERR_INVALID_ARGUMENT, "tiles or out is NULL"),
    (_tb, dict(out=TL + 64), fastvr.ERR_INVALID_ARGUMENT, "out overlaps tiles"),
    (_tb, dict(Wg=1 << 27, C=64), fastvr.ERR_UNSUPPORTED, "2^31"),
])
def test_tile_rejects(lib, fn, kw, status, needle):
    assert fn(**kw) == status
    assert needle in fastvr.last_error()


@pytest.mark.parametrize("kw,needle", [
    (dict(z=None), "z_lq is NULL"),
    (dict(z=Z + 4), "8-byte aligned"),
    (dict(sigma=float("nan")), "sigma"),
    (dict(out=Z + 16), "out overlaps z_lq"),
])
def test_tile_blend_update_rejects(lib, kw, needle):
    assert _tb(update=True, **kw) == fastvr.ERR_INVALID_ARGUMENT
    assert needle in fastvr.last_error()


@pytest.mark.parametrize("kw", [dict(B=0), dict(T=0), dict(Hg=0), dict(C=0)])
def test_tile_empty_is_ok(lib, kw):
    assert _tg(**kw) == fastvr.OK
    assert _tb(**kw) == fastvr.OK
    assert _tb(update=True, **kw) == fastvr.OK


def test_valid_calls_reach_the_launcher(lib):
    """Valid arguments pass every check and reach the launcher.  Runs only
    against the host-only build whose launchers are stand-ins that launch
    nothing (tests/host_stubs.cpp, built by tests/test_host_sanitizers.py), so
    the fake addresses are never used; the real library is skipped."""
    if not hasattr(lib, "fastvr_stub_launch_count"):
        pytest.skip("needs the host-only build with stand-in launchers")
    lib.fastvr_stub_launch_count.restype = ctypes.c_int64
    calls = [
        lambda: _fwd(),
        lambda: _fwd(d=128, window_chunks=1, Nkv=200, chunk_len=64),
        lambda: _fwd(lse=None, q_chunk_offset=2, Nq=16, Nkv=64),
        lambda: _fwd_ex(),
        lambda: _fwd_ex(o_bf16=1, o_st=136, o_sb=64 * 136, k_sb=100 * 128, v_sb=100 * 128, Nkv=100),
        lambda: _app(),
        lambda: _app(B=3, d=128, cache_len=0, n_new=100),
        lambda: _ring(),
        lambda: _ring(chunk_index=0, window_chunks=0, n_new=5, chunk_len=64),
        lambda: _ring(d=64, chunk_len=72, n_new=72, chunk_index=9, window_chunks=7),
        lambda: _bwd(),
        lambda: _bwd(d=128, Nq=16, Nkv=64, q_chunk_offset=3, window_chunks=1),
        lambda: _bwd(Nq=0, q=None, dout=None, o=None, dq=None, lse=None, rs=None),
        lambda: _bwd_na(),
        lambda: _bwd_na(H=64, Nq=65536, Nkv=65536, d=128),
        lambda: _os(),
        lambda: _os(out=Z, out_bf16=1),
        lambda: _tg(),
        lambda: _tb(),
        lambda: _tb(update=True),
    ]
    for i, call in enumerate(calls):
        before = lib.fastvr_stub_launch_count()
        assert call() == fastvr.OK, (i, fastvr.last_error())
        assert fastvr.last_error() == ""
        assert lib.fastvr_stub_launch_count() == before + 1, i


def test_error_is_thread_local(lib):
    import threading
    assert _fwd(d=96) == fastvr.ERR_UNSUPPORTED
    seen = {}

    def other():
        seen["msg"] = fastvr.last_error()
    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen["msg"] == ""
    assert "head_dim" in fastvr.last_error()


def test_wrapper_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(fastvr, "_LIB", None)
    monkeypatch.setattr(fastvr, "LIB_PATH", "/nonexistent/libfastvr.so")
    with pytest.raises(RuntimeError, match="missing"):
        fastvr.load()


def test_input_generator_is_deterministic():
    from paper_2609_36757_amd import workloads
    a = workloads.make_qkv(1, 33, 40, 2, 64, seed=9)
    b = workloads.make_qkv(1, 33, 40, 2, 64, seed=9)
    c = workloads.make_qkv(1, 33, 40, 2, 64, seed=10)
    for x, y in zip(a, b):
        assert x.dtype == workloads.torch.bfloat16
        assert workloads.torch.equal(x, y)
    assert not workloads.torch.equal(a[0], c[0])


def test_workload_registry_shapes():
    from paper_2609_36757_amd import workloads
    w = workloads.WORKLOADS
    assert (w["1080p"].n_tokens, w["1080p"].chunk_len, w["1080p"].n_chunks) == (65280, 16320, 4)
    assert (w["480p"].n_tokens, w["480p"].chunk_len, w["480p"].n_chunks) == (18720, 3120, 6)
    assert (w["wide_sw"].n_tokens, w["wide_sw"].window_chunks, w["wide_sw"].n_chunks) == (138720, 2, 9)
    assert w["1080p_stream"].stream_chunk == 3 and w["1080p_stream"].seed == w["1080p"].seed
    assert w["tiny"].d == 64 and w["tiny"].scale == 0.125


def test_c_client_compiles_and_runs(lib, tmp_path):
    """The header compiles as strict C99 and a C program linked against the
    library gets the same host-side results (tests/c_abi_client.c)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    here = os.path.dirname(os.path.abspath(__file__))
    libdir = os.path.dirname(fastvr.LIB_PATH)
    exe = str(tmp_path / "c_abi_client")
    cmd = [cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.dirname(HEADER),
           os.path.join(here, "c_abi_client.c"), "-o", exe, f"-L{libdir}", "-lfastvr", f"-Wl,-rpath,{libdir}",
           "-Wl,--allow-shlib-undefined"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
