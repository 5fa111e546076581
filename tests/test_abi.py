"""The C ABI without a GPU: the library loads, exports every function that
include/acsc.h declares, and rejects bad arguments on the host (before any
HIP call, so these run on a machine without a GPU)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "acsc.h")
LIB = os.path.join(ROOT, "paper_2609_14339_amd", "libacsc.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z][a-z0-9_]*)\s*\([^;{]*\)\s*;", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libacsc.so is not built (run __graft_entry__.build())")
    return C.CDLL(LIB)


def test_header_declares_the_four_hot_path_calls():
    fns = declared_functions()
    for name in ("ac_mask_pack", "ac_unpack_scatter", "sc_build_prior", "sc_correct"):
        assert name in fns


def test_library_exports_every_declared_function(lib):
    fns = declared_functions()
    assert len(fns) >= 8
    for name in fns:
        assert hasattr(lib, name), name


def test_python_binding_names_match_the_header():
    import paper_2609_14339_amd as pk
    assert set(pk.EXPORTED) == set(declared_functions())
    for name in pk.EXPORTED:
        if not name.startswith("acsc_"):
            assert callable(getattr(pk, name)), name


class Key(C.Structure):
    _fields_ = [("seed", C.c_uint64), ("step", C.c_uint64), ("layer", C.c_uint32),
                ("microbatch", C.c_uint32), ("B", C.c_uint32), ("S", C.c_uint32),
                ("H", C.c_uint32)]


def _err(lib):
    lib.acsc_last_error.restype = C.c_char_p
    return lib.acsc_last_error().decode()


def test_keep_count_on_host(lib):
    k = C.c_int(0)
    lib.ac_keep_count.argtypes = [C.c_int, C.c_double, C.POINTER(C.c_int)]
    assert lib.ac_keep_count(2048, 0.05, C.byref(k)) == 0 and k.value == 102
    assert lib.ac_keep_count(8192, 0.02, C.byref(k)) == 0 and k.value == 164
    assert lib.ac_keep_count(10, 0.01, C.byref(k)) == -1 and "outside" in _err(lib)
    assert lib.ac_keep_count(70000, 0.5, C.byref(k)) == -1


def test_pack_and_unpack_reject_bad_arguments_before_launch(lib):
    vp = C.c_void_p
    lib.ac_mask_pack.argtypes = [vp, C.c_int, C.c_int64, C.c_int, C.c_int64, C.c_int,
                                 C.POINTER(Key), vp, vp, vp]
    lib.ac_unpack_scatter.argtypes = [vp, vp, C.c_int, C.c_int64, C.c_int, C.c_int,
                                      C.POINTER(Key), C.c_float, vp, C.c_int64, vp]
    key = Key(seed=1, step=1, layer=0, microbatch=0, B=2, S=4, H=64)
    fake = vp(0x1000)
    # wrong dtype, K out of range, shape mismatch with the key, ld too small,
    # null pointers, misaligned pointers
    assert lib.ac_mask_pack(fake, 7, 8, 64, 64, 4, C.byref(key), fake, None, None) == -2
    assert lib.ac_mask_pack(fake, 1, 8, 64, 64, 0, C.byref(key), fake, None, None) == -1
    assert lib.ac_mask_pack(fake, 1, 8, 64, 64, 65, C.byref(key), fake, None, None) == -1
    assert lib.ac_mask_pack(fake, 1, 9, 64, 64, 4, C.byref(key), fake, None, None) == -1
    assert "key.B*key.S" in _err(lib)
    assert lib.ac_mask_pack(fake, 1, 8, 64, 63, 4, C.byref(key), fake, None, None) == -1
    assert lib.ac_mask_pack(None, 1, 8, 64, 64, 4, C.byref(key), fake, None, None) == -1
    assert lib.ac_mask_pack(fake, 1, 8, 64, 64, 4, None, fake, None, None) == -1
    assert lib.ac_mask_pack(vp(0x1001), 1, 8, 64, 64, 4, C.byref(key), fake, None, None) == -3
    assert lib.ac_mask_pack(vp(0x1002), 0, 8, 64, 64, 4, C.byref(key), fake, None, None) == -3
    assert lib.ac_unpack_scatter(fake, None, 1, 8, 64, 4, C.byref(key), 1.0, fake, 32, None) == -1
    assert lib.ac_unpack_scatter(fake, None, 1, 8, 64, 4, C.byref(key), float("inf"), fake, 64,
                                 None) == -1
    assert lib.ac_unpack_scatter(fake, vp(0x1003), 1, 8, 64, 4, C.byref(key), 1.0, fake, 64,
                                 None) == -3
    # zero rows is a no-op that succeeds without touching any pointer
    key0 = Key(seed=1, step=1, layer=0, microbatch=0, B=0, S=4, H=64)
    assert lib.ac_mask_pack(None, 1, 0, 64, 64, 4, C.byref(key0), None, None, None) == 0
    assert lib.ac_unpack_scatter(None, None, 1, 0, 64, 4, C.byref(key0), 1.0, None, 64, None) == 0


def test_psgd_workspace_and_rejects_bad_arguments_before_launch(lib):
    import paper_2609_14339_amd as pk
    vp = C.c_void_p
    b = C.c_size_t(0)
    assert lib.psgd_workspace_size(8192, 28672, 99, 1, C.byref(b)) == 0
    big = b.value
    # the bf16 copy of M dominates: at least m * n * 2 bytes
    assert big >= 8192 * 28672 * 2
    assert lib.psgd_workspace_size(256, 256, 8, 0, C.byref(b)) == 0 and b.value < big
    assert lib.psgd_workspace_size(64, 64, 65, 1, C.byref(b)) == -1 and "r=65" in _err(lib)
    assert lib.psgd_workspace_size(64, 64, 8, 5, C.byref(b)) == -2
    fake = 0x10000

    def mat(**kw):
        d = dict(G=fake, E=fake, P=fake, Q=fake, out=fake, m=64, n=48, ws=fake, ws_bytes=1 << 30)
        d.update(kw)
        return pk.PsgdMatrix(**d)

    def call(name, mats, r=4, dt=1):
        arr = (pk.PsgdMatrix * len(mats))(*mats)
        return getattr(lib, name)(len(mats), arr, dt, r, None)

    for name in ("psgd_project", "psgd_orthogonalize", "psgd_decompress", "psgd_step"):
        assert call(name, [mat()], r=0) == -1
        assert call(name, [mat()], r=49) == -1            # r > min(m, n)
        assert call(name, [mat()], dt=3) == -2
        assert call(name, [mat(ws_bytes=1024)]) == -5      # ACSC_ENOSPC
        assert call(name, [mat(ws=fake + 16)]) == -3       # workspace alignment
        assert call(name, [mat(E=fake + 4)]) == -3         # E 16-byte alignment
        assert call(name, [mat(P=None)]) == -1
        assert call(name, [mat(), mat(m=0)]) == -1         # every matrix checked first
        assert "matrix 1" in _err(lib)
    assert call("psgd_project", [mat(G=None)]) == -1
    assert call("psgd_project", [mat(G=fake + 2)]) == -3
    assert call("psgd_decompress", [mat(out=None)]) == -1
    assert call("psgd_decompress", [mat(out=fake + 1)]) == -3
    assert call("psgd_step", [mat(G=None)]) == -1
    # an empty call succeeds without touching anything; a negative count is rejected
    assert lib.psgd_project(0, None, 1, 4, None) == 0
    assert lib.psgd_step(-1, None, 1, 4, None) == -1


def test_batched_mask_calls_reject_bad_arguments_before_launch(lib):
    vp, i64 = C.c_void_p, C.c_int64
    lib.ac_mask_pack_batched.argtypes = [vp, C.c_int, C.c_int, i64, C.c_int, i64, i64, C.c_int, C.POINTER(Key),
                                         vp, i64, vp, vp, i64, vp]
    lib.ac_unpack_scatter_batched.argtypes = [vp, i64, C.c_int, C.c_int, i64, C.c_int, C.c_int, C.POINTER(Key),
                                              vp, vp, i64, C.c_float, vp, i64, i64, vp]
    key = Key(seed=1, step=1, layer=0, microbatch=0, B=2, S=4, H=64)
    f = vp(0x10000)
    rows, H, K = 8, 64, 4
    pack = lambda nl, xs, vs, ii, io, istr, k=key: lib.ac_mask_pack_batched(
        f, 1, nl, rows, H, H, xs, K, C.byref(k), f, vs, ii, io, istr, None)
    unpack = lambda nl, vs, ii, io, istr, ys, k=key: lib.ac_unpack_scatter_batched(
        f, vs, 1, nl, rows, H, K, C.byref(k), ii, io, istr, 1.0, f, H, ys, None)
    assert pack(-1, 0, 0, None, None, 0) == -1
    assert pack(65536, 0, 0, None, None, 0) == -1
    assert pack(3, rows * H, rows * K - 1, None, None, 0) == -1 and "overlap" in _err(lib)
    assert pack(3, rows * H, rows * K, None, f, rows * K - 1) == -1
    assert pack(3, -1, rows * K, None, None, 0) == -1
    assert pack(1, 0, 0, f, f, 0) == -1 and "exclusive" in _err(lib)
    big = Key(seed=1, step=1, layer=0xFFFFFFFF, microbatch=0, B=2, S=4, H=64)
    assert pack(2, rows * H, rows * K, None, None, 0, big) == -1 and "layer" in _err(lib)
    assert pack(1, 0, 0, vp(0x10001), None, 0) == -3
    assert unpack(3, rows * K, None, None, 0, rows * H - 1) == -1 and "overlap" in _err(lib)
    assert unpack(3, rows * K, None, f, rows * K - 1, rows * H) == -1
    assert unpack(2, rows * K, f, f, rows * K, rows * H) == -1
    assert unpack(1, 0, None, vp(0x10001), 0, 0) == -3
    # no boundaries, or no rows: a no-op that touches no pointer
    assert lib.ac_mask_pack_batched(None, 1, 0, rows, H, H, 0, K, C.byref(key), None, 0, None, None, 0, None) == 0
    key0 = Key(seed=1, step=1, layer=0, microbatch=0, B=0, S=4, H=64)
    assert lib.ac_unpack_scatter_batched(None, 0, 1, 5, 0, H, K, C.byref(key0), None, None, 0, 1.0, None, H, 0,
                                         None) == 0


def test_static_correction_rejects_bad_arguments_before_launch(lib):
    vp = C.c_void_p
    lib.sc_correct_static.argtypes = [vp, C.c_int, C.c_int, C.c_int, vp, vp, vp, C.c_int, C.c_float, vp, vp]
    f = vp(0x10000)
    assert lib.sc_correct_static(f, 1, 64, 64, f, f, f, 0, 0.3, f, None) == -1
    assert lib.sc_correct_static(f, 9, 64, 64, f, f, f, 4, 0.3, f, None) == -2
    # beyond the static scratch: refused on the host with ACSC_ENOSPC
    assert lib.sc_correct_static(f, 1, 65536, 8192, f, f, f, 128, 0.3, f, None) == -5
    assert "scratch" in _err(lib)


def test_stats_filter_takes_a_name_or_null_on_host(lib):
    # no launch happens: the filter is host state only
    lib.acsc_stats_only.argtypes = [C.c_char_p]
    assert lib.acsc_stats_only(b"sc_ema") == 0
    assert lib.acsc_stats_only(b"x" * 64) == -1 and "64" in _err(lib)
    assert lib.acsc_stats_only(None) == 0
    assert lib.acsc_stats_only(b"") == 0
