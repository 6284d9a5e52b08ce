"""Host-side checks of the C ABI: the library loads, exports every declared entry point, sizes its buffers like the
documented format, and rejects invalid arguments before any HIP call. CPU only (no compute call)."""
import ctypes
import os
import re
import struct

import numpy as np
import pytest

from oracle import format_oracle as fmt
from synth import LayerSpec

fb = pytest.importorskip("paper_2608_15602_amd.fluxbin")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(fb.LIB_PATH):
        pytest.fail("libfluxbin.so is not built; run `python -m paper_2608_15602_amd.build`")
    return fb.lib()


def _declared_functions():
    with open(os.path.join(ROOT, "include", "fluxbin.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(fluxbin_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function(L):
    names = _declared_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(fb.EXPORTS)


def test_status_strings(L):
    for s in range(5):
        assert L.fluxbin_status_string(s)
    assert L.fluxbin_status_string(99) == b"unknown status"


def _shape(**kw):
    base = dict(M=4096, N=4096, Kb=2, Ks=1, mu=8, g_r=128, S=82, g_s=82)
    base.update(kw)
    return fb.make_shape(**base)


def _spec(sh):
    return LayerSpec("q", M=sh.M, N=sh.N, Kb=sh.Kb, Ks=sh.Ks, mu=sh.mu, S=sh.S, g_r=sh.g_r, g_s=sh.g_s)


@pytest.mark.parametrize("kw", [
    {}, dict(M=28672, N=8192, Kb=3, S=410, g_s=410), dict(M=8192, N=28672, Kb=3, S=1434, g_s=1434),
    dict(M=512, N=256, mu=4, S=8, g_s=8), dict(M=1, N=1, Kb=1, Ks=0, S=0, g_r=1, g_s=1),
    dict(M=70, N=300, Kb=4, Ks=2, S=300, g_s=128, g_r=256), dict(M=65, N=100, S=0, g_r=100),
    dict(Ks=2, S=256, g_s=8), dict(Ks=2, S=512, g_s=16), dict(g_r=64, Ks=2, S=256, g_s=8),
    dict(M=70, N=300, Kb=3, S=40, g_r=64, g_s=16), dict(M=512, N=256, mu=4, S=64, g_s=4, g_r=32),
])
def test_pack_query_matches_format(L, kw):
    sh = _shape(**kw)
    assert fb.fluxbin_pack_query(sh) == fmt.packed_bytes(_spec(sh))["total"]


@pytest.mark.parametrize("kw,status", [
    (dict(M=0), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(M=(1 << 27) + 1), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(N=0), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(N=70000, g_r=70000), fb.FLUXBIN_ERR_UNSUPPORTED),
    (dict(Kb=0), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(Kb=5), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(Ks=-1), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(mu=0), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(mu=6), fb.FLUXBIN_ERR_UNSUPPORTED),
    (dict(g_r=0), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(g_r=100), fb.FLUXBIN_ERR_INVALID_ARG),       # not whole sub-vectors of mu = 8
    (dict(g_r=96), fb.FLUXBIN_ERR_UNSUPPORTED),        # whole sub-vectors, but neither a divisor nor a multiple of 128
    (dict(S=5000), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(S=300, g_s=12), fb.FLUXBIN_ERR_INVALID_ARG),
    (dict(S=300, g_s=192), fb.FLUXBIN_ERR_UNSUPPORTED),
])
def test_pack_query_rejects(L, kw, status):
    n = ctypes.c_size_t(123)
    st = L.fluxbin_pack_query(ctypes.byref(_shape(**kw)), ctypes.byref(n))
    assert st == status
    assert L.fluxbin_last_error_message()
    assert n.value == 123


def test_pack_query_null(L):
    assert L.fluxbin_pack_query(None, None) == fb.FLUXBIN_ERR_INVALID_ARG


def _host_weights(sh, sal_idx):
    W = (sh.N + 31) // 32
    Gr = -(-sh.N // sh.g_r)
    Gs = -(-sh.S // sh.g_s) if sh.S else 0
    arrs = dict(
        signs=np.zeros((sh.Kb, sh.M, W), np.uint32), alpha_r=np.zeros((sh.Kb, sh.M, Gr), np.uint16),
        alpha_c=np.zeros((sh.Kb, sh.N), np.uint16), sal_idx=np.asarray(sal_idx, np.int32),
        sal_signs=np.zeros((sh.Ks, sh.M, W), np.uint32), alpha_sr=np.zeros((sh.Ks, sh.M, max(Gs, 1)), np.uint16),
        alpha_sc=np.zeros((sh.Ks, sh.N), np.uint16))
    w = fb.Weights(*(arrs[k].ctypes.data for k in ("signs", "alpha_r", "alpha_c", "sal_idx", "sal_signs",
                                                     "alpha_sr", "alpha_sc")), 0)
    return w, arrs


FAKE_DEVICE_PTR = 0x7F0000001000   # never dereferenced: every case below fails validation first


@pytest.mark.parametrize("sal,status", [
    ([3, 2, 10, 11], fb.FLUXBIN_ERR_INVALID_ARG),        # not increasing
    ([1, 1, 10, 11], fb.FLUXBIN_ERR_INVALID_ARG),        # duplicate
    ([1, 2, 10, 300], fb.FLUXBIN_ERR_INVALID_ARG),       # out of range (N = 256)
    ([-1, 2, 10, 11], fb.FLUXBIN_ERR_INVALID_ARG),
])
def test_pack_rejects_bad_salient_set(L, sal, status):
    sh = fb.make_shape(64, 256, 2, 1, 8, 128, 4, 4)
    w, keep = _host_weights(sh, sal)
    n = fb.fluxbin_pack_query(sh)
    out = fb.Layer()
    st = L.fluxbin_pack(ctypes.byref(sh), ctypes.byref(w), FAKE_DEVICE_PTR, n, ctypes.byref(out), None)
    assert st == status
    assert b"sal_idx" in L.fluxbin_last_error_message()


def test_pack_rejects_small_buffer_and_nulls(L):
    sh = fb.make_shape(64, 256, 2, 1, 8, 128, 4, 4)
    w, keep = _host_weights(sh, [1, 2, 3, 4])
    n = fb.fluxbin_pack_query(sh)
    out = fb.Layer()
    assert L.fluxbin_pack(ctypes.byref(sh), ctypes.byref(w), FAKE_DEVICE_PTR, n - 1, ctypes.byref(out), None) == \
        fb.FLUXBIN_ERR_BUFFER_TOO_SMALL
    assert L.fluxbin_pack(ctypes.byref(sh), ctypes.byref(w), None, n, ctypes.byref(out), None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_pack(ctypes.byref(sh), None, FAKE_DEVICE_PTR, n, ctypes.byref(out), None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    w.alpha_c = None
    assert L.fluxbin_pack(ctypes.byref(sh), ctypes.byref(w), FAKE_DEVICE_PTR, n, ctypes.byref(out), None) == \
        fb.FLUXBIN_ERR_INVALID_ARG


def _header_bytes(spec):
    """The 256-byte header as documented in include/fluxbin.h, written independently of the library."""
    d = fmt.derived(spec)
    pb = fmt.packed_bytes(spec)
    h = struct.pack("<II", fmt.MAGIC, fmt.VERSION)
    h += struct.pack("<qqiiiiqqq", spec.M, spec.N, spec.Kb, spec.Ks, spec.mu, 0, spec.g_r, spec.S, spec.g_s)
    h += struct.pack("<8q", d["Npad"], d["Sv"], d["NC"], d["NSC"], d["Mp"], d["Gr"], d["Gs"], d["NRP"])
    h += struct.pack("<7Q", pb["off_signs"], pb["off_rscale"], pb["off_colscale"], pb["off_xidx"],
                     pb["off_chunk_plane"], pb["off_sal_idx"], pb["total"])
    return h + bytes(256 - len(h))


def _fake_layer(L, spec):
    hdr = _header_bytes(spec)
    out = fb.Layer()
    total = fmt.packed_bytes(spec)["total"]
    st = L.fluxbin_layer_from_header(ctypes.create_string_buffer(hdr, 256), FAKE_DEVICE_PTR, total, ctypes.byref(out))
    assert st == 0, L.fluxbin_last_error_message()
    return out, total


@pytest.mark.parametrize("g_r,g_s", [(128, 17), (64, 8)])
def test_layer_from_header(L, g_r, g_s):
    spec = LayerSpec("h", M=1000, N=300, Kb=3, Ks=1, mu=8, S=17, g_r=g_r, g_s=g_s)
    out, total = _fake_layer(L, spec)
    pb = fmt.packed_bytes(spec)
    d = fmt.derived(spec)
    assert out.off_signs == pb["off_signs"] and out.off_sal_idx == pb["off_sal_idx"]
    assert out.NSC == d["NSC"] and out.Mp == d["Mp"] and out.NRP == d["NRP"]
    assert out.format_version == fb.FORMAT_VERSION == 2 and out.bytes == total
    bad = bytearray(_header_bytes(spec))
    bad[0] ^= 1
    assert L.fluxbin_layer_from_header(ctypes.create_string_buffer(bytes(bad), 256), FAKE_DEVICE_PTR, total,
                                       ctypes.byref(fb.Layer())) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_layer_from_header(ctypes.create_string_buffer(_header_bytes(spec), 256), FAKE_DEVICE_PTR,
                                       total - 1, ctypes.byref(fb.Layer())) == fb.FLUXBIN_ERR_BUFFER_TOO_SMALL


def test_gemv_rejects_bad_arguments(L):
    spec = LayerSpec("h", M=1000, N=300, Kb=2, Ks=1, mu=8, S=17, g_r=128, g_s=17)
    lay, _ = _fake_layer(L, spec)
    X, Y, WS = 0x7F0000100000, 0x7F0000200000, 0x7F0000300000
    g = L.fluxbin_lut_gemv
    assert g(None, X, Y, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert g(ctypes.byref(lay), None, Y, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert g(ctypes.byref(lay), X, None, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert g(ctypes.byref(lay), X, Y, 2, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert g(ctypes.byref(lay), X, X + 100, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG   # x/y overlap
    gb = L.fluxbin_lut_gemm_smallbatch
    assert gb(ctypes.byref(lay), 0, X, 300, Y, 1000, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert gb(ctypes.byref(lay), 8193, X, 300, Y, 1000, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert gb(ctypes.byref(lay), -1, X, 300, Y, 1000, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert gb(ctypes.byref(lay), 2, X, 299, Y, 1000, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert gb(ctypes.byref(lay), 2, X, 300, Y, 999, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_stream_probe(ctypes.byref(lay), X, 1000, None) == fb.FLUXBIN_ERR_BUFFER_TOO_SMALL
    # a descriptor edited by hand no longer matches its shape
    lay.off_signs += 256
    assert g(ctypes.byref(lay), X, Y, 0, WS, 1 << 20, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_workspace_init(None, 16, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_workspace_init(WS, 6, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_debug_indices(None, X, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_unpack_canonical(None, X, None, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_stream_probe(None, X, 1024, None) == fb.FLUXBIN_ERR_INVALID_ARG


def test_decomposition_sizes_and_bad_arguments(L):
    """Workspace of the decomposition (int8 signs, then the column-scale partial sums of up to 64 row slices of at
    least 256 rows) and argument checks that fail before any launch."""
    n = ctypes.c_size_t(0)
    assert L.fluxbin_rc_workspace_query(1000, 300, 3, ctypes.byref(n)) == fb.FLUXBIN_OK
    signs = 3 * 1000 * 300
    assert n.value == ((signs + 255) // 256) * 256 + 3 * 2 * 300 * 8   # 1000 // 256 = 3 slices
    assert L.fluxbin_rc_workspace_query(100, 300, 1, ctypes.byref(n)) == fb.FLUXBIN_OK
    assert n.value == ((100 * 300 + 255) // 256) * 256 + 1 * 2 * 300 * 8
    assert L.fluxbin_rc_workspace_query(100000, 10, 1, ctypes.byref(n)) == fb.FLUXBIN_OK
    assert n.value == ((100000 * 10 + 255) // 256) * 256 + 64 * 2 * 10 * 8
    assert L.fluxbin_rc_workspace_query(0, 300, 1, ctypes.byref(n)) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_rc_workspace_query(10, 300, 5, ctypes.byref(n)) == fb.FLUXBIN_ERR_INVALID_ARG
    assert L.fluxbin_rc_workspace_query(10, 300, 1, None) == fb.FLUXBIN_ERR_INVALID_ARG
    X, S, A, C, WS = 0x7F0000100000, 0x7F0000200000, 0x7F0000300000, 0x7F0000400000, 0x7F0000500000
    d = L.fluxbin_rc_decompose
    ok_ws = 1 << 30
    assert d(None, None, None, None, None, 0, 1, 64, 256, 2, 3, 128, 1e-12, S, A, C, WS, ok_ws, None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    assert d(X, None, None, None, None, 0, 1, 64, 256, 2, -1, 128, 1e-12, S, A, C, WS, ok_ws, None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    assert d(X, None, None, None, None, 0, 1, 64, 256, 2, 3, 0, 1e-12, S, A, C, WS, ok_ws, None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    assert d(X, None, None, None, None, 0, 1, 64, 256, 2, 3, 128, float("nan"), S, A, C, WS, ok_ws, None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    assert d(X, None, None, None, None, 0, 1, 64, 256, 2, 3, 128, -1.0, S, A, C, WS, ok_ws, None) == \
        fb.FLUXBIN_ERR_INVALID_ARG
    assert d(X, None, None, None, None, 0, 1, 64, 256, 2, 3, 128, 1e-12, S, A, C, WS, 100, None) == \
        fb.FLUXBIN_ERR_BUFFER_TOO_SMALL
    assert d(X, None, S, None, C, 2, 128, 64, 256, 2, 3, 128, 1e-12, S, A, C, WS, ok_ws, None) == \
        fb.FLUXBIN_ERR_INVALID_ARG   # prior signs without their row scales
    ss = L.fluxbin_structural_search
    assert ss(None, A, 64, 256, 128, 8, C, S, None, None) == fb.FLUXBIN_ERR_INVALID_ARG
    assert ss(X, A, 64, 256, 2048, 8, C, S, None, None) == fb.FLUXBIN_ERR_UNSUPPORTED   # group > 1024
    assert ss(X, A, 64, 256, 128, 200, C, S, None, None) == fb.FLUXBIN_ERR_INVALID_ARG  # s > g
    assert ss(X, A, 64, 256, 128, 0, C, S, None, None) == fb.FLUXBIN_ERR_INVALID_ARG


def test_tuning_is_explicit_process_state(L):
    """The launch-plan tuning is read from the environment once and otherwise changed only by fluxbin_set_tuning; the
    context manager restores the previous values."""
    t0 = fb.fluxbin_get_tuning()
    assert set(t0) == {n for n, _ in fb.Tuning._fields_}
    with fb.tuning(mfma=0, nt=512):
        t1 = fb.fluxbin_get_tuning()
        assert t1["mfma"] == 0 and t1["nt"] == 512
    assert fb.fluxbin_get_tuning() == t0
    fb.fluxbin_set_tuning(None)
    d = fb.fluxbin_get_tuning()
    assert d["mfma"] == -1 and d["min_units"] == -1 and d["early"] == -1 and d["mfma_r2"] == 1 and d["bat_r2"] == 1
    fb.fluxbin_set_tuning(t0)
    with pytest.raises(KeyError):
        with fb.tuning(no_such_field=1):
            pass
    assert L.fluxbin_get_tuning(None) == fb.FLUXBIN_ERR_INVALID_ARG


def test_plan_query_and_noalloc_validate_on_the_host(L):
    info = fb.PlanInfo()
    assert L.fluxbin_plan_query(None, 1, ctypes.byref(info)) == fb.FLUXBIN_ERR_INVALID_ARG
    X = ctypes.c_void_p(1 << 20)
    Y = ctypes.c_void_p(1 << 24)
    assert L.fluxbin_lut_gemv_noalloc(None, X, Y, 0, None) == fb.FLUXBIN_ERR_INVALID_ARG


def test_random_shapes_and_headers_are_rejected_cleanly(L):
    """Random shapes through fluxbin_pack_query and random or corrupted 256-byte headers through
    fluxbin_layer_from_header: every call returns a status (the host-sanitizer test runs this under ASan/UBSan)."""
    rng = np.random.default_rng(5)
    n = ctypes.c_size_t(0)
    for _ in range(2000):
        vals = rng.integers(-3, 1 << 17, size=8)
        sh = fb.make_shape(int(vals[0]), int(vals[1]), int(vals[2] % 7) - 1, int(vals[3] % 7) - 1,
                           int(vals[4] % 10), int(vals[5]), int(vals[6]), int(vals[7]))
        st = L.fluxbin_pack_query(ctypes.byref(sh), ctypes.byref(n))
        assert st in (fb.FLUXBIN_OK, fb.FLUXBIN_ERR_INVALID_ARG, fb.FLUXBIN_ERR_UNSUPPORTED)
        if st == fb.FLUXBIN_OK:
            assert n.value == fmt.packed_bytes(_spec(sh))["total"]
    good = _header_bytes(LayerSpec("h", M=100, N=300, Kb=2, Ks=1, mu=8, S=20, g_r=64, g_s=8))
    for k in range(500):
        h = bytearray(good)
        for _ in range(int(rng.integers(1, 6))):
            h[int(rng.integers(0, 256))] = int(rng.integers(0, 256))
        if k % 50 == 0:
            h = bytearray(rng.integers(0, 256, size=256, dtype=np.uint8).tobytes())
        st = L.fluxbin_layer_from_header(ctypes.create_string_buffer(bytes(h), 256), FAKE_DEVICE_PTR, 1 << 40,
                                         ctypes.byref(fb.Layer()))
        assert st in (fb.FLUXBIN_OK, fb.FLUXBIN_ERR_INVALID_ARG, fb.FLUXBIN_ERR_UNSUPPORTED,
                      fb.FLUXBIN_ERR_BUFFER_TOO_SMALL)
