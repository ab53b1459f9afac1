"""The C ABI library loads, exports every declared entry point, and rejects bad arguments
on the host before launching anything.  No kernel runs here (no GPU needed): every call
below either fails validation or is a documented no-op (rows == 0)."""

import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "nestquant.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nq_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2502_09720_amd as nq
    return nq.library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"nq_encode", "nq_decode", "nq_matmul"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_sizes(lib):
    assert lib.nq_codes_words(3, 64) == 24
    assert lib.nq_beta_words(3, 64) == 3
    assert lib.nq_beta_words(3, 128) == 3
    assert lib.nq_beta_words(3, 136) == 6
    assert lib.nq_codes_words(3, 12) == -1
    assert lib.nq_codes_words(-1, 64) == -1


def test_status_strings(lib):
    for s in range(4):
        assert lib.nq_status_string(s)
    assert lib.nq_version() >= 100


def _p(q=14, k=4, base=None):
    from paper_2502_09720_amd.binding import _Params
    return _Params(q, k, 10.0 / (max(k, 1) * max(q, 1)) if base is None else base)


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: each call below fails validation
NULL = ctypes.c_void_p(0)
S = ctypes.c_void_p(0)


def _pd(decoder, strategy=0):
    p = _p()
    p.decoder, p.strategy = decoder, strategy
    return p


def _pm(mult, k=4, q=14):
    p = _p(q=q, k=k)
    for i, m in enumerate(mult):
        p.mult[i] = m
    return p


@pytest.mark.parametrize("case", [
    dict(p=_pd(2)), dict(p=_pd(-1)), dict(p=_pd(0, 2)), dict(p=_pd(0, -1)),
    dict(p=_pm((1, 2, 2, 3))), dict(p=_pm((3, 2, 4, 5))), dict(p=_pm((1, 2, 3, 65))),
    dict(p=_pm((0, 1, 2, 3))), dict(p=_pm((1, 2, 3, 4), k=3)), dict(p=_pm((2, 3, 0, 0), k=3)),
    dict(p=_pm((-1, 2, 3, 4))),
    dict(p=None), dict(p=_p(q=1)), dict(p=_p(q=17)), dict(p=_p(k=0)), dict(p=_p(k=5)),
    dict(p=_p(base=0.0)), dict(p=_p(base=-1.0)), dict(p=_p(base=float("nan"))),
    dict(p=_p(base=1e-9)), dict(cols=12), dict(cols=0), dict(cols=65544), dict(rows=-1),
    dict(ld=32), dict(x=NULL), dict(codes=NULL), dict(x=ctypes.c_void_p(0x1004)),
    dict(dtype=7),
])
def test_encode_rejects(lib, case):
    p = case.get("p", _p())
    args = dict(rows=4, cols=64, ld=64, x=FAKE, codes=FAKE, dtype=0)
    args.update(case)
    pp = None if p is None else ctypes.byref(p)
    st = lib.nq_encode(pp, args["x"], args["dtype"], args["rows"], args["cols"], args["ld"],
                       args["codes"], FAKE, FAKE, S)
    assert st in (1, 2)
    assert lib.nq_last_error()


def test_encode_zero_rows_is_noop(lib):
    p = _p()
    assert lib.nq_encode(ctypes.byref(p), NULL, 0, 0, 64, 64, NULL, NULL, NULL, S) == 0


@pytest.mark.parametrize("case", [
    dict(p=_p(q=0)), dict(cols=7), dict(ld=8), dict(out=NULL), dict(dtype=3),
    dict(out=ctypes.c_void_p(0x1002)), dict(rows=-5),
])
def test_decode_rejects(lib, case):
    p = case.get("p", _p())
    args = dict(rows=4, cols=64, ld=64, out=FAKE, dtype=0)
    args.update(case)
    st = lib.nq_decode(ctypes.byref(p), FAKE, FAKE, FAKE, args["rows"], args["cols"],
                       args["out"], args["dtype"], args["ld"], S)
    assert st in (1, 2)


@pytest.mark.parametrize("case", [
    dict(pa=_p(k=9)), dict(pw=_p(q=99)), dict(K=20), dict(M=-1), dict(ldc=3), dict(c=NULL),
])
def test_matmul_rejects(lib, case):
    pa, pw = case.get("pa", _p()), case.get("pw", _p())
    args = dict(M=4, N=8, K=64, ldc=8, c=FAKE)
    args.update(case)
    st = lib.nq_matmul(ctypes.byref(pa), FAKE, FAKE, FAKE, args["M"], ctypes.byref(pw), FAKE,
                       FAKE, FAKE, args["N"], args["K"], args["c"], args["ldc"], S)
    assert st == 1


def test_workspace_size(lib):
    assert lib.nq_matmul_workspace_size(16, 4096, 4096) == 16 * 4096 * 2   # skinny: A tile
    assert lib.nq_matmul_workspace_size(0, 4096, 4096) == 0
    ws = lib.nq_matmul_workspace_size(2048, 4096, 4096)
    assert ws >= (2048 + 4096) * 4096 * 2                          # bf16 tiles of A and W
    assert lib.nq_matmul_workspace_size(100, 10, 12) == -1


def test_matmul_ex_rejects_small_workspace(lib):
    p = _p()
    need = lib.nq_matmul_workspace_size(300, 200, 64)
    assert need > 0
    st = lib.nq_matmul_ex(ctypes.byref(p), FAKE, FAKE, FAKE, 300, ctypes.byref(p), FAKE, FAKE,
                          FAKE, 200, 64, FAKE, 200, FAKE, need - 16, S)
    assert st == 1
    st = lib.nq_matmul_ex(ctypes.byref(p), FAKE, FAKE, FAKE, 300, ctypes.byref(p), FAKE, FAKE,
                          FAKE, 200, 64, FAKE, 200, NULL, need, S)
    assert st == 1


@pytest.mark.parametrize("stages", [0, 4, 8, 11, -1])
def test_matmul_stages_rejects_bad_mask(lib, stages):
    p = _p()
    need = lib.nq_matmul_workspace_size(300, 200, 64)
    st = lib.nq_matmul_stages(stages, ctypes.byref(p), FAKE, FAKE, FAKE, 300, ctypes.byref(p),
                              FAKE, FAKE, FAKE, 200, 64, FAKE, 200, FAKE, need, S)
    assert st == 1
    assert b"stages" in lib.nq_last_error()


def test_matmul_stages_validates_like_ex(lib):
    p = _p()
    need = lib.nq_matmul_workspace_size(300, 200, 64)
    for stages in (1, 2, 3):
        st = lib.nq_matmul_stages(stages, ctypes.byref(p), FAKE, FAKE, FAKE, 300,
                                  ctypes.byref(p), FAKE, FAKE, FAKE, 200, 64, FAKE, 200, FAKE,
                                  need - 16, S)
        assert st == 1
        st = lib.nq_matmul_stages(stages, ctypes.byref(p), FAKE, FAKE, FAKE, 300,
                                  ctypes.byref(p), FAKE, FAKE, FAKE, 200, 64, FAKE, 100, FAKE,
                                  need, S)
        assert st == 1


@pytest.mark.parametrize("q,k,ok", [(14, 4, True), (15, 4, True), (16, 4, False),
                                    (16, 3, True), (8, 4, True), (12, 4, True)])
def test_matmul_int8_needs_small_kq(lib, q, k, ok):
    """k * q <= 63 keeps |t X2| <= 2 k q within int8; larger products are refused.  M = 0, so
    an accepted call returns before any launch."""
    good, test = _p(), _p(q=q, k=k)
    for pa, pw in ((good, test), (test, good)):
        st = lib.nq_matmul_stages(7, ctypes.byref(pa), FAKE, FAKE, FAKE, 0, ctypes.byref(pw),
                                  FAKE, FAKE, FAKE, 200, 64, FAKE, 200, FAKE, 0, S)
        assert st == (0 if ok else 2)
        if not ok:
            assert b"int8" in lib.nq_last_error()


@pytest.mark.parametrize("q,mult,ok", [(16, (1, 2, 3), True), (16, (1, 2, 4), False),
                                       (7, (2, 5, 9), True), (7, (2, 5, 10), False),
                                       (2, (10, 20, 31), True), (2, (10, 20, 32), False)])
def test_matmul_int8_needs_small_multiples(lib, q, mult, ok):
    """With a beta table the int8 bound is 2q * mult_k <= 127 (|m X2| <= 2q m)."""
    good, test = _p(), _pm(mult, k=len(mult), q=q)
    for pa, pw in ((good, test), (test, good)):
        st = lib.nq_matmul_stages(7, ctypes.byref(pa), FAKE, FAKE, FAKE, 0, ctypes.byref(pw),
                                  FAKE, FAKE, FAKE, 200, 64, FAKE, 200, FAKE, 0, S)
        assert st == (0 if ok else 2)


def test_matmul_empty_is_noop(lib):
    p = _p()
    assert lib.nq_matmul(ctypes.byref(p), NULL, NULL, NULL, 0, ctypes.byref(p), NULL, NULL,
                         NULL, 5, 64, NULL, 5, S) == 0


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    import paper_2502_09720_amd.binding as b
    monkeypatch.setenv("NESTQUANT_LIB", str(tmp_path / "missing.so"))
    monkeypatch.setattr(b, "_LIB", None)
    with pytest.raises(RuntimeError):
        b.library()


def test_params_layout():
    """nq_params is {int32 q, int32 k, double base, int32 decoder, int32 strategy,
    int32 mult[4]}: 40 bytes, base at offset 8, decoder at 16, strategy at 20, mult at 24."""
    from paper_2502_09720_amd.binding import _Params
    assert ctypes.sizeof(_Params) == 40
    assert _Params.base.offset == 8 and _Params.decoder.offset == 16
    assert _Params.strategy.offset == 20 and _Params.mult.offset == 24


@pytest.mark.parametrize("case", [
    dict(cols=24), dict(cols=11008), dict(cols=65536), dict(cols=4), dict(dtype=5),
    dict(rows=-1), dict(ld=8), dict(y=NULL), dict(x=ctypes.c_void_p(0x1004)),
    dict(y=ctypes.c_void_p(0x1000)),                 # y overlaps x
])
def test_rotate_rejects(lib, case):
    args = dict(rows=4, cols=64, ld=64, x=FAKE, y=ctypes.c_void_p(0x100000), dtype=0)
    args.update(case)
    st = lib.nq_rotate(args["x"], args["dtype"], args["rows"], args["cols"], args["ld"],
                       args["y"], args["ld"] if args["ld"] >= 64 else 64, S)
    assert st in (1, 2)
    assert lib.nq_last_error()


def test_rotate_zero_rows_is_noop(lib):
    assert lib.nq_rotate(NULL, 0, 0, 4096, 4096, NULL, 4096, S) == 0
    assert lib.nq_rotate(NULL, 0, 0, 14336, 14336, NULL, 14336, S) == 0


def _betas(vals):
    return (ctypes.c_double * len(vals))(*vals)


@pytest.mark.parametrize("case", [
    dict(q=1), dict(q=17), dict(decoder=2), dict(m=0), dict(m=65), dict(n=-1),
    dict(n=1 << 31), dict(betas=None), dict(vals=(0.1, 0.1)), dict(vals=(0.2, 0.1)),
    dict(vals=(0.0, 0.1)), dict(vals=(float("inf"),)), dict(vals=(float("nan"), 1.0)),
    dict(v=NULL), dict(mse=NULL), dict(v=ctypes.c_void_p(0x1004)),
])
def test_beta_stats_rejects(lib, case):
    args = dict(q=16, decoder=0, v=FAKE, n=10, vals=(0.1, 0.2, 0.3), mse=FAKE)
    args.update(case)
    vals = args["vals"]
    m = case.get("m", len(vals))
    b = None if "betas" in case else _betas(vals + (1.0,) * max(0, m - len(vals)))
    st = lib.nq_beta_stats(args["q"], args["decoder"], args["v"], args["n"], b, m, args["mse"],
                           FAKE, S)
    assert st == 1


def test_beta_stats_empty_is_noop(lib):
    assert lib.nq_beta_stats(16, 0, NULL, 0, _betas((0.1, 0.2)), 2, NULL, NULL, S) == 0


@pytest.mark.parametrize("case", [
    dict(m=0), dict(m=65), dict(k=0), dict(k=5), dict(n=-1), dict(mse=NULL), dict(chosen=NULL),
    dict(loss=NULL), dict(ws=NULL), dict(ws_bytes=8), dict(ws=ctypes.c_void_p(0x1004)),
])
def test_beta_dp_rejects(lib, case):
    args = dict(mse=FAKE, n=10, m=4, k=2, chosen=FAKE, loss=FAKE, ws=FAKE, ws_bytes=1 << 20)
    args.update(case)
    st = lib.nq_beta_dp(args["mse"], FAKE, args["n"], args["m"], args["k"], args["chosen"],
                        args["loss"], args["ws"], args["ws_bytes"], S)
    assert st == 1


def test_beta_dp_workspace_size(lib):
    f = lib.nq_beta_dp_workspace_size
    f.argtypes = [ctypes.c_int64, ctypes.c_int32]
    f.restype = ctypes.c_int64
    q = lambda m: m * (m + 1) // 2 + m             # transition costs and overload counts
    assert f(0, 4) == 2 * q(4) * 8                 # one level-2 node and one level-3 node
    assert f(1 << 18, 50) == (64 + 1) * q(50) * 8  # 2^18 samples: 64 nodes of 4096
    assert f(-1, 4) == -1 and f(10, 0) == -1 and f(10, 65) == -1


# Every entry point that takes no workspace must not allocate: the library imports no
# allocation routine from the HIP runtime at all.
ALLOCATORS = re.compile(r"^(hip(Ext)?Malloc\w*|hipFree\w*|hipHostMalloc|hipHostAlloc|"
                        r"hipMallocAsync|hipMallocFromPoolAsync|hipMemPool\w*|hipArrayCreate|"
                        r"hipMalloc3D\w*)$")


def test_library_imports_no_allocator(lib):
    import shutil
    import subprocess
    import paper_2502_09720_amd as nq
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--undefined-only", nq.library_path()], capture_output=True,
                         text=True, check=True).stdout
    imported = {line.split()[-1].split("@")[0] for line in out.splitlines() if line.strip()}
    assert "hipLaunchKernel" in imported                       # the listing is the real one
    assert not {name for name in imported if ALLOCATORS.match(name)}


@pytest.mark.parametrize("case", [
    dict(flags=1), dict(flags=2), dict(flags=16), dict(flags=8), dict(pa=None), dict(x=NULL),
    dict(K=12),
    dict(dtype=9), dict(c=NULL), dict(ldc=10), dict(ws_bytes=0),
    dict(pa=_p(q=16)),                              # int8 needs k q <= 63
])
def test_encode_matmul_rejects(lib, case):
    p = _p()
    args = dict(flags=0, pa=p, x=FAKE, dtype=0, M=300, K=64, c=FAKE, ldc=200, ws_bytes=1 << 30)
    args.update(case)
    if "pa" in case and case["pa"] is not None and case["pa"].q == 16:
        args["flags"] = 4
    pa = None if args["pa"] is None else ctypes.byref(args["pa"])
    st = lib.nq_encode_matmul(args["flags"], pa, args["x"], args["dtype"], args["M"], args["K"],
                              args["K"], FAKE, FAKE, FAKE, ctypes.byref(p), FAKE, FAKE, FAKE,
                              200, args["c"], args["ldc"], FAKE, args["ws_bytes"], S)
    assert st in (1, 2)


def test_encode_matmul_empty_is_noop(lib):
    p = _p()
    assert lib.nq_encode_matmul(0, ctypes.byref(p), NULL, 0, 0, 64, 64, NULL, NULL, NULL,
                                ctypes.byref(p), NULL, NULL, NULL, 0, NULL, 0, NULL, 0, S) == 0


@pytest.mark.parametrize("case,status", [
    (dict(cols=2048), 2), (dict(cols=4104), 2), (dict(cols=32768), 2), (dict(cols=28672), 2),
    (dict(strategy=1), 2), (dict(q=1), 1), (dict(x=NULL), 1), (dict(ld=100), 1),
    (dict(dtype=7), 2), (dict(x=ctypes.c_void_p(0x1004)), 1),
])
def test_rotate_encode_rejects(lib, case, status):
    """Widths the in-LDS rotation does not hold, Opt-beta, and the checks of nq_encode."""
    args = dict(cols=4096, strategy=0, q=14, x=FAKE, ld=None, dtype=2)
    args.update(case)
    p = _pd(0, args["strategy"])
    p.q = args["q"]
    ld = args["ld"] if args["ld"] is not None else args["cols"]
    st = lib.nq_rotate_encode(ctypes.byref(p), args["x"], args["dtype"], 4, args["cols"], ld,
                              FAKE, FAKE, FAKE, S)
    assert st == status
    assert lib.nq_last_error()


def test_rotate_encode_zero_rows_is_noop(lib):
    p = _p()
    for cols in (3584, 4096, 7168, 8192, 14336, 16384):
        assert lib.nq_rotate_encode(ctypes.byref(p), NULL, 2, 0, cols, cols, NULL, NULL, NULL,
                                    S) == 0
