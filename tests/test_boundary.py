"""The C-ABI boundary without a GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flashkmeans.h")
LIB = os.path.join(ROOT, "paper_2608_12629_amd", "libflashkmeans.so")

OK, EINVAL, EUNSUP, EWS, EHIP, ESCRATCH = 0, -1, -2, -3, -4, -5
SCRATCH_BYTES = 64 << 20
F32, BF16, F16 = 0, 1, 2


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kmeans_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} not built (run __graft_entry__.build())")
    L = ctypes.CDLL(LIB)
    i64, i32, vp, sz = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
    L.kmeans_workspace_bytes.argtypes = [i64, i64, i64, i64, i32]
    L.kmeans_workspace_bytes.restype = sz
    L.kmeans_assign.argtypes = [vp, i32, vp, i64, i64, i64, i64, vp, vp, vp, sz, vp]
    L.kmeans_update.argtypes = [vp, i32, vp, vp, i64, i64, i64, i64, vp, vp, vp, sz, vp]
    L.kmeans_lloyd.argtypes = [vp, i32, vp, i64, i64, i64, i64, i32, vp, vp, vp, vp, vp, sz, vp]
    L.kmeans_lloyd_noalloc.argtypes = [vp, i32, vp, i64, i64, i64, i64, i32, vp, vp, vp, vp, vp]
    L.kmeans_knn_workspace_bytes.argtypes = [i64, i64, i64, i64, i32, i32]
    L.kmeans_knn_workspace_bytes.restype = sz
    L.kmeans_knn.argtypes = [vp, vp, i32, i64, i64, i64, i64, i32, vp, vp, vp, sz, vp]
    L.kmeans_status_string.argtypes = [ctypes.c_int]
    L.kmeans_status_string.restype = ctypes.c_char_p
    return L


def test_header_declares_the_calls():
    assert declared_functions() == ["kmeans_assign", "kmeans_knn", "kmeans_knn_workspace_bytes",
                                    "kmeans_lloyd", "kmeans_lloyd_noalloc",
                                    "kmeans_status_string", "kmeans_update",
                                    "kmeans_workspace_bytes"]
    text = open(HEADER).read()
    assert re.search(r"#define KMEANS_SCRATCH_BYTES \(\(size_t\)64 << 20\)", text)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for st in (OK, EINVAL, EUNSUP, EWS, EHIP, ESCRATCH):
        s = lib.kmeans_status_string(st).decode()
        assert s and s != "unknown status"
    assert lib.kmeans_status_string(12345).decode() == "unknown status"


def test_workspace_bytes(lib):
    ws = lambda B, N, D, K, dt=BF16: lib.kmeans_workspace_bytes(B, N, D, K, dt)
    assert ws(1, 8_388_608, 128, 4096) > 0
    assert ws(1, 1000, 64, 10, F32) > 0
    # a workspace sized for N serves every smaller N (same B, D, K), on both
    # update paths (sorted: K = 1024; per-chunk partials: K = 64)
    for K in (1024, 64):
        prev = 0
        for N in (1, 100, 2048, 2049, 4096, 4097, 65536, 1 << 20):
            cur = ws(1, N, 128, K)
            assert cur >= prev
            prev = cur
    # the small-K one-hot path (16-bit, D = 64, K = 64)
    prev = 0
    for N in (1, 100, 2048, 2049, 4096, 65536, 1 << 20):
        cur = ws(2, N, 64, 64, F16)
        assert cur >= prev
        prev = cur
    # fp32 workgroups shrink for small problems (more of them): still monotone
    for D, K in ((64, 256), (128, 4096)):
        prev = 0
        for N in (1, 65536, 65537, 131071, 131072, 262143, 262144, 1 << 20):
            cur = ws(1, N, D, K, F32)
            assert cur >= prev, (D, K, N)
            prev = cur
    for K in (1, 7, 64, 1000, 4096, 32768, 65536):
        assert ws(1, 65536, 64, K) > 0
    assert ws(4, 1000, 64, 10) >= ws(1, 1000, 64, 10)
    # rejected shapes report 0
    assert ws(0, 10, 64, 4) == 0 and ws(1, 0, 64, 4) == 0 and ws(1, 10, 64, 0) == 0
    for D in (1, 3, 40, 100, 250, 272, 300, 2047):
        assert ws(1, 1000, D, 10) > 0, D    # served on zero-padded rows
    assert ws(1, 1000, 40, 10) > ws(1, 1000, 48, 10)  # plus the padded copies
    for D in (3, 17, 255):
        assert ws(1, 1000, D, 10, F32) > 0, D
    assert ws(1, 1000, 272, 10, F32) == 0   # fp32 rows past 256
    assert ws(1, 1000, 2049, 10) == 0
    for D in (16, 48, 96, 160, 208, 256, 288, 384, 640, 992, 2048):
        assert ws(1, 1000, D, 10) > 0, D    # 16-bit shapes in the domain
    for D in (16, 48, 80, 112, 128, 144, 256):
        assert ws(1, 1000, D, 10, F32) > 0, D
    assert ws(1, 10, 64, 70000) == 0        # K above the sort limit
    assert ws(1, 10, 64, 4, 7) == 0         # unknown dtype


FAKE = 0x10000          # a non-null, 16-byte-aligned address that is never dereferenced


def _assign(lib, X=FAKE, dt=BF16, C=FAKE, B=1, N=100, D=64, K=4, idx=FAKE, md=FAKE,
            ws=FAKE, wsb=1 << 40):
    return lib.kmeans_assign(X, dt, C, B, N, D, K, idx, md, ws, wsb, None)


def _update(lib, X=FAKE, dt=BF16, idx=FAKE, Cp=FAKE, B=1, N=100, D=64, K=4, Co=FAKE, n=FAKE,
            ws=FAKE, wsb=1 << 40):
    return lib.kmeans_update(X, dt, idx, Cp, B, N, D, K, Co, n, ws, wsb, None)


def _lloyd(lib, X=FAKE, dt=BF16, C=FAKE, B=1, N=100, D=64, K=4, iters=3, idx=FAKE, md=FAKE,
           n=FAKE, obj=None, ws=FAKE, wsb=1 << 40):
    return lib.kmeans_lloyd(X, dt, C, B, N, D, K, iters, idx, md, n, obj, ws, wsb, None)


@pytest.mark.parametrize("call", [_assign, _update, _lloyd])
def test_rejections_before_any_device_call(lib, call):
    assert call(lib, X=None) == EINVAL
    assert call(lib, X=FAKE + 4) == EINVAL          # misaligned
    assert call(lib, dt=3) == EINVAL
    assert call(lib, B=0) == EINVAL
    assert call(lib, N=0) == EINVAL
    assert call(lib, N=-5) == EINVAL
    assert call(lib, K=0) == EINVAL
    assert call(lib, D=0) == EINVAL
    assert call(lib, D=4096) == EUNSUP
    assert call(lib, D=2049) == EUNSUP
    assert call(lib, dt=F32, D=272) == EUNSUP  # fp32 rows up to 256
    assert call(lib, K=70000) == EUNSUP
    assert call(lib, N=1 << 31) == EUNSUP
    assert call(lib, ws=None) == EWS
    assert call(lib, wsb=16) == EWS


def test_specific_rejections(lib):
    assert _assign(lib, C=None) == EINVAL
    assert _assign(lib, idx=None) == EINVAL
    assert _assign(lib, md=None) == EINVAL
    assert _update(lib, idx=None) == EINVAL
    assert _update(lib, Cp=None) == EINVAL
    assert _update(lib, Co=None) == EINVAL
    assert _update(lib, n=None) == EINVAL
    assert _lloyd(lib, iters=0) == EINVAL
    assert _lloyd(lib, n=None) == EINVAL
    assert _lloyd(lib, obj=FAKE + 8) == EINVAL
    exact = lib.kmeans_workspace_bytes(1, 100, 64, 4, BF16)
    assert _assign(lib, wsb=exact - 1) == EWS


def _noalloc(lib, X=FAKE, dt=BF16, C=FAKE, B=1, N=100, D=64, K=4, iters=3, idx=FAKE, md=FAKE,
             n=FAKE, obj=None):
    return lib.kmeans_lloyd_noalloc(X, dt, C, B, N, D, K, iters, idx, md, n, obj, None)


def test_noalloc_rejections_before_any_device_call(lib):
    """The static-scratch entry point validates like kmeans_lloyd and rejects
    problems whose workspace exceeds the array, all before touching a GPU."""
    assert _noalloc(lib, X=None) == EINVAL
    assert _noalloc(lib, C=FAKE + 4) == EINVAL
    assert _noalloc(lib, n=None) == EINVAL
    assert _noalloc(lib, obj=FAKE + 8) == EINVAL
    assert _noalloc(lib, iters=0) == EINVAL
    assert _noalloc(lib, dt=3) == EINVAL
    assert _noalloc(lib, D=4096) == EUNSUP
    assert _noalloc(lib, K=70000) == EUNSUP
    # the 8M-point workload needs ~138 MiB of workspace: too big for the array
    assert lib.kmeans_workspace_bytes(1, 8_388_608, 128, 4096, BF16) > SCRATCH_BYTES
    assert _noalloc(lib, N=8_388_608, D=128, K=4096) == ESCRATCH
    # the largest N that fits, and the first that does not (fp32, D = 64, K = 256)
    fits = lambda N: lib.kmeans_workspace_bytes(1, N, 64, 256, F32) <= SCRATCH_BYTES
    lo, hi = 1, 1 << 28
    while hi - lo > 1:
        mid = (lo + hi) // 2
        lo, hi = (mid, hi) if fits(mid) else (lo, mid)
    assert _noalloc(lib, dt=F32, N=hi, D=64, K=256) == ESCRATCH
    assert fits(65536)   # the fp32 blob workload fits


def test_binding_refuses_without_library(tmp_path, monkeypatch):
    """The Python binding raises instead of falling back when the library is absent."""
    import importlib
    import paper_2608_12629_amd.kmeans as km
    monkeypatch.setattr(km, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        km._load()
    importlib.reload(km)  # restore the module state with the real library


def _knn(lib, Q=FAKE, R=FAKE, dt=BF16, B=1, M=50, N=100, D=64, k=5, ni=FAKE, nd=FAKE, ws=FAKE,
         wsb=1 << 40):
    return lib.kmeans_knn(Q, R, dt, B, M, N, D, k, ni, nd, ws, wsb, None)


def test_knn_rejections(lib):
    assert _knn(lib, Q=None) == EINVAL
    assert _knn(lib, R=FAKE + 8) == EINVAL
    assert _knn(lib, ni=None) == EINVAL
    assert _knn(lib, nd=None) == EINVAL
    assert _knn(lib, k=0) == EINVAL
    assert _knn(lib, k=101) == EINVAL         # k > N
    assert _knn(lib, M=0) == EINVAL
    assert _knn(lib, dt=3) == EINVAL
    assert _knn(lib, dt=F32) == EUNSUP        # fp32 search not built
    assert _knn(lib, D=272) == EUNSUP
    assert _knn(lib, k=33) == EUNSUP
    assert _knn(lib, ws=None) == EWS
    assert _knn(lib, wsb=16) == EWS
    kw = lambda **a: lib.kmeans_knn_workspace_bytes(*[a.get(n, v) for n, v in
                                                      (("B", 1), ("M", 50), ("N", 100), ("D", 64),
                                                       ("k", 5), ("dt", BF16))])
    assert kw() > 0 and kw(k=33) == 0 and kw(dt=F32) == 0
    assert kw(N=1000) >= kw(N=100)


def test_calibration_library_exports_its_header():
    """libfkm_calib.so (the benchmark's in-run ceilings) exports every call that
    include/fkm_calib.h declares and rejects bad arguments on the host."""
    path = os.path.join(ROOT, "paper_2608_12629_amd", "libfkm_calib.so")
    if not os.path.exists(path):
        pytest.fail(f"{path} not built (run __graft_entry__.build())")
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "fkm_calib.h")).read(),
                  flags=re.S)
    names = sorted(set(re.findall(r"\b(fkm_calib_\w+)\s*\(", text)))
    assert names == ["fkm_calib_gather", "fkm_calib_mfma", "fkm_calib_read"]
    L = ctypes.CDLL(path)
    for n in names:
        assert hasattr(L, n), n
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    L.fkm_calib_mfma.argtypes = [vp, i32, i32, vp]
    L.fkm_calib_read.argtypes = [vp, sz, vp, i32, vp]
    L.fkm_calib_gather.argtypes = [vp, i64, i32, vp, i64, vp, i32, vp]
    assert L.fkm_calib_mfma(None, 512, 10, None) == -1
    assert L.fkm_calib_mfma(FAKE, 0, 10, None) == -1
    assert L.fkm_calib_read(FAKE, 17, FAKE, 16, None) == -1        # not whole 16-byte chunks
    assert L.fkm_calib_read(FAKE + 4, 16, FAKE, 16, None) == -1    # misaligned
    assert L.fkm_calib_gather(FAKE, 10, 2048, FAKE, 10, FAKE, 16, None) == -1  # rows > 1 KiB
    assert L.fkm_calib_gather(FAKE, 0, 256, FAKE, 10, FAKE, 16, None) == -1
