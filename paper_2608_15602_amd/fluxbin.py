"""Thin ctypes binding of libfluxbin (include/fluxbin.h): argument marshalling only.

Every step of the hot path runs in the library's HIP kernels; PyTorch only provides device memory and the stream.
The functions keep the C names. Tensors must be on the current CUDA (HIP) device unless stated otherwise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
# FLUXBIN_LIBRARY selects another build of the same library (the host-sanitizer build of the CPU tests)
LIB_PATH = os.environ.get("FLUXBIN_LIBRARY") or os.path.join(HERE, "libfluxbin.so")

FLUXBIN_OK = 0
FLUXBIN_ERR_INVALID_ARG = 1
FLUXBIN_ERR_UNSUPPORTED = 2
FLUXBIN_ERR_BUFFER_TOO_SMALL = 3
FLUXBIN_ERR_HIP = 4
FORMAT_VERSION = 2
HEADER_BYTES = 256

# Entry points declared in include/fluxbin.h.
EXPORTS = (
    "fluxbin_status_string", "fluxbin_last_error_message", "fluxbin_pack_query", "fluxbin_pack",
    "fluxbin_layer_from_header", "fluxbin_workspace_query", "fluxbin_workspace_init", "fluxbin_lut_gemv",
    "fluxbin_lut_gemm_smallbatch", "fluxbin_debug_indices", "fluxbin_unpack_canonical", "fluxbin_stream_probe",
    "fluxbin_rc_workspace_query", "fluxbin_rc_decompose", "fluxbin_structural_search", "fluxbin_get_tuning",
    "fluxbin_set_tuning", "fluxbin_plan_query", "fluxbin_lut_gemv_noalloc",
)
NOALLOC_SCRATCH_BYTES = 8 << 20

KERNEL_NAMES = {0: "batch1", 1: "generic", 2: "lut_batch", 3: "mfma", 4: "rows", 5: "mfma_rows"}


class FluxbinError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"fluxbin status {status}: {message}")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("Kb", ctypes.c_int32), ("Ks", ctypes.c_int32),
                ("mu", ctypes.c_int32), ("reserved0", ctypes.c_int32), ("g_r", ctypes.c_int64),
                ("S", ctypes.c_int64), ("g_s", ctypes.c_int64)]


class Weights(ctypes.Structure):
    _fields_ = [("signs", ctypes.c_void_p), ("alpha_r", ctypes.c_void_p), ("alpha_c", ctypes.c_void_p),
                ("sal_idx", ctypes.c_void_p), ("sal_signs", ctypes.c_void_p), ("alpha_sr", ctypes.c_void_p),
                ("alpha_sc", ctypes.c_void_p), ("inputs_on_device", ctypes.c_int32)]


class Layer(ctypes.Structure):
    _fields_ = [("shape", Shape), ("d_base", ctypes.c_void_p), ("bytes", ctypes.c_uint64),
                ("format_version", ctypes.c_uint32), ("reserved1", ctypes.c_uint32),
                ("Npad", ctypes.c_int64), ("Sv", ctypes.c_int64), ("NC", ctypes.c_int64), ("NSC", ctypes.c_int64),
                ("Mp", ctypes.c_int64), ("Gr", ctypes.c_int64), ("Gs", ctypes.c_int64), ("NRP", ctypes.c_int64),
                ("off_signs", ctypes.c_uint64), ("off_rscale", ctypes.c_uint64), ("off_colscale", ctypes.c_uint64),
                ("off_xidx", ctypes.c_uint64), ("off_chunk_plane", ctypes.c_uint64), ("off_sal_idx", ctypes.c_uint64)]


class Tuning(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("nt", "min_units", "blocks", "blocks_per_cu", "depth", "mfma_depth",
                                             "early", "rpt", "mfma", "generic", "mfma_r2", "bat_r2", "rows",
                                             "batch_tile", "mfma_rows", "align", "big_units")]


class PlanInfo(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("threads", ctypes.c_int32), ("rows_per_tile", ctypes.c_int32),
                ("depth", ctypes.c_int32), ("batch_groups", ctypes.c_int32),
                ("second_kernel_reduction", ctypes.c_int32), ("early", ctypes.c_int32), ("batch_tiles", ctypes.c_int32),
                ("batch_tile_rows", ctypes.c_int32), ("workgroups_per_tile", ctypes.c_int32),
                ("tiles", ctypes.c_int64), ("units", ctypes.c_int64), ("workgroups", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_uint64)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libfluxbin.so (built by ``python -m paper_2608_15602_amd.build``). Raises if it is missing: there is no
    fallback implementation."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FluxbinError(-1, f"{LIB_PATH} is missing; build it with `python -m paper_2608_15602_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.fluxbin_status_string.restype = ctypes.c_char_p
        L.fluxbin_status_string.argtypes = [ctypes.c_int]
        L.fluxbin_last_error_message.restype = ctypes.c_char_p
        L.fluxbin_last_error_message.argtypes = []
        L.fluxbin_pack_query.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(sz)]
        L.fluxbin_pack.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(Weights), vp, sz, ctypes.POINTER(Layer), vp]
        L.fluxbin_layer_from_header.argtypes = [vp, vp, sz, ctypes.POINTER(Layer)]
        L.fluxbin_workspace_query.argtypes = [ctypes.POINTER(Layer), i32, ctypes.POINTER(sz)]
        L.fluxbin_workspace_init.argtypes = [vp, sz, vp]
        L.fluxbin_lut_gemv.argtypes = [ctypes.POINTER(Layer), vp, vp, i32, vp, sz, vp]
        L.fluxbin_lut_gemm_smallbatch.argtypes = [ctypes.POINTER(Layer), i32, vp, i64, vp, i64, i32, vp, sz, vp]
        L.fluxbin_debug_indices.argtypes = [ctypes.POINTER(Layer), vp, vp]
        L.fluxbin_unpack_canonical.argtypes = [ctypes.POINTER(Layer), vp, vp, vp]
        L.fluxbin_stream_probe.argtypes = [ctypes.POINTER(Layer), vp, sz, vp]
        L.fluxbin_rc_workspace_query.argtypes = [i64, i64, i32, ctypes.POINTER(sz)]
        L.fluxbin_rc_decompose.argtypes = [vp, vp, vp, vp, vp, i32, i64, i64, i64, i32, i32, i64, ctypes.c_double,
                                           vp, vp, vp, vp, sz, vp]
        L.fluxbin_structural_search.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, vp]
        L.fluxbin_get_tuning.argtypes = [ctypes.POINTER(Tuning)]
        L.fluxbin_set_tuning.argtypes = [ctypes.POINTER(Tuning)]
        L.fluxbin_plan_query.argtypes = [ctypes.POINTER(Layer), i32, ctypes.POINTER(PlanInfo)]
        L.fluxbin_lut_gemv_noalloc.argtypes = [ctypes.POINTER(Layer), vp, vp, i32, vp]
        for name in EXPORTS:
            if name not in ("fluxbin_status_string", "fluxbin_last_error_message"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != FLUXBIN_OK:
        msg = lib().fluxbin_last_error_message().decode(errors="replace")
        raise FluxbinError(status, msg or lib().fluxbin_status_string(status).decode())


def make_shape(M, N, Kb, Ks, mu, g_r, S, g_s) -> Shape:
    return Shape(int(M), int(N), int(Kb), int(Ks), int(mu), 0, int(g_r), int(S), int(g_s))


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return int(stream) if not hasattr(stream, "cuda_stream") else stream.cuda_stream


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if hasattr(t, "data_ptr"):
        return t.data_ptr()
    return t.ctypes.data  # numpy array (host inputs)


def fluxbin_pack_query(shape: Shape) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().fluxbin_pack_query(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


class PackedLayer:
    """A packed device buffer (torch uint8 tensor) and its C descriptor."""

    def __init__(self, buf, layer: Layer):
        self.buf = buf
        self.layer = layer

    @property
    def shape(self) -> Shape:
        return self.layer.shape


def fluxbin_pack(shape: Shape, weights: Dict[str, object], stream=None, device=None) -> PackedLayer:
    """Pack canonical weights. ``weights`` maps the fluxbin_weights field names to torch tensors on the device (or to
    numpy arrays in host memory, then all of them must be numpy)."""
    import torch
    nbytes = fluxbin_pack_query(shape)
    on_dev = all(hasattr(v, "data_ptr") for v in weights.values() if v is not None)
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device or "cuda")
    keep = {k: (v.contiguous() if hasattr(v, "contiguous") else v) for k, v in weights.items()}
    w = Weights(_ptr(keep.get("signs")), _ptr(keep.get("alpha_r")), _ptr(keep.get("alpha_c")),
                _ptr(keep.get("sal_idx")), _ptr(keep.get("sal_signs")), _ptr(keep.get("alpha_sr")),
                _ptr(keep.get("alpha_sc")), 1 if on_dev else 0)
    out = Layer()
    _check(lib().fluxbin_pack(ctypes.byref(shape), ctypes.byref(w), buf.data_ptr(), nbytes, ctypes.byref(out),
                              _stream(stream)))
    return PackedLayer(buf, out)


def fluxbin_layer_from_header(header: bytes, buf) -> PackedLayer:
    out = Layer()
    hb = ctypes.create_string_buffer(bytes(header[:HEADER_BYTES]), HEADER_BYTES)
    _check(lib().fluxbin_layer_from_header(hb, buf.data_ptr(), buf.numel(), ctypes.byref(out)))
    return PackedLayer(buf, out)


def fluxbin_workspace_query(layer: PackedLayer, B: int = 1) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().fluxbin_workspace_query(ctypes.byref(layer.layer), int(B), ctypes.byref(n)))
    return n.value


def fluxbin_workspace_init(ws, stream=None) -> None:
    _check(lib().fluxbin_workspace_init(ws.data_ptr(), ws.numel() * ws.element_size(), _stream(stream)))


def make_workspace(layer: PackedLayer, B: int = 1, stream=None):
    """Allocate (torch) and zero-fill (library kernel) a workspace for batch B."""
    import torch
    n = fluxbin_workspace_query(layer, B)
    ws = torch.empty(max(256, (n + 255) // 256 * 256), dtype=torch.uint8, device=layer.buf.device)
    fluxbin_workspace_init(ws, stream)
    return ws


def _check_io(layer: PackedLayer, x, y, out_fp32: bool, B: int) -> None:
    """The library takes raw pointers: dtype, device, length and inner stride are checked here, before the call."""
    import torch
    s = layer.shape
    dev = layer.buf.device
    if x.dtype != torch.float16 or x.device != dev or x.stride(-1) != 1:
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, f"x must be fp16 on {dev} with unit inner stride")
    if x.shape[-1] < s.N or (x.dim() == 2 and x.shape[0] < B):
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, f"x has shape {tuple(x.shape)}, needs [{B}, >= {s.N}]")
    want = torch.float32 if out_fp32 else torch.float16
    if y.dtype != want or y.device != dev or y.stride(-1) != 1:
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, f"y must be {want} on {dev} with unit inner stride")
    if y.shape[-1] < s.M or (y.dim() == 2 and y.shape[0] < B):
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, f"y has shape {tuple(y.shape)}, needs [{B}, >= {s.M}]")


def fluxbin_lut_gemv(layer: PackedLayer, x, y=None, out_fp32: bool = False, workspace=None, stream=None):
    import torch
    M = layer.shape.M
    if y is None:
        y = torch.empty(M, dtype=torch.float32 if out_fp32 else torch.float16, device=x.device)
    if x.dim() != 1 or y.dim() != 1:
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, "fluxbin_lut_gemv takes one activation vector x [N] and y [M]")
    _check_io(layer, x, y, out_fp32, 1)
    if workspace is None:
        workspace = make_workspace(layer, 1, stream)
    _check(lib().fluxbin_lut_gemv(ctypes.byref(layer.layer), x.data_ptr(), y.data_ptr(), 1 if out_fp32 else 0,
                                  workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))
    return y


def fluxbin_lut_gemv_noalloc(layer: PackedLayer, x, y, out_fp32: bool = False, stream=None):
    """fluxbin_lut_gemv without a workspace (the library's static device scratch); y must be preallocated."""
    if x.dim() != 1 or y.dim() != 1:
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, "fluxbin_lut_gemv_noalloc takes x [N] and y [M]")
    _check_io(layer, x, y, out_fp32, 1)
    _check(lib().fluxbin_lut_gemv_noalloc(ctypes.byref(layer.layer), x.data_ptr(), y.data_ptr(), 1 if out_fp32 else 0,
                                          _stream(stream)))
    return y


def fluxbin_lut_gemm_smallbatch(layer: PackedLayer, x, y=None, out_fp32: bool = False, workspace=None, stream=None):
    """x: fp16 [B, N] (row stride x.stride(0)); returns y [B, M]."""
    import torch
    B = x.shape[0]
    M = layer.shape.M
    if y is None:
        y = torch.empty(B, M, dtype=torch.float32 if out_fp32 else torch.float16, device=x.device)
    if x.dim() != 2 or y.dim() != 2:
        raise FluxbinError(FLUXBIN_ERR_INVALID_ARG, "fluxbin_lut_gemm_smallbatch takes x [B, N] and y [B, M]")
    _check_io(layer, x, y, out_fp32, B)
    if workspace is None:
        workspace = make_workspace(layer, B, stream)
    _check(lib().fluxbin_lut_gemm_smallbatch(ctypes.byref(layer.layer), int(B), x.data_ptr(), int(x.stride(0)),
                                             y.data_ptr(), int(y.stride(0)), 1 if out_fp32 else 0,
                                             workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                             _stream(stream)))
    return y


def fluxbin_debug_indices(layer: PackedLayer, stream=None):
    import torch
    s = layer.shape
    n = (2 * layer.layer.NSC) * s.M * (128 // s.mu)
    out = torch.empty(n, dtype=torch.uint8, device=layer.buf.device)
    _check(lib().fluxbin_debug_indices(ctypes.byref(layer.layer), out.data_ptr(), _stream(stream)))
    return out.view(2 * layer.layer.NSC, s.M, 128 // s.mu)


def fluxbin_unpack_canonical(layer: PackedLayer, stream=None) -> Tuple[object, object]:
    import torch
    s = layer.shape
    W = (s.N + 31) // 32
    signs = torch.empty(s.Kb * s.M * W, dtype=torch.int32, device=layer.buf.device)
    dense = None
    if s.S > 0 and s.Ks > 0:
        dense = torch.empty(s.Ks * s.M * ((s.S + 31) // 32), dtype=torch.int32, device=layer.buf.device)
    _check(lib().fluxbin_unpack_canonical(ctypes.byref(layer.layer), signs.data_ptr(),
                                          dense.data_ptr() if dense is not None else None, _stream(stream)))
    return signs.view(s.Kb, s.M, W), (dense.view(s.Ks, s.M, -1) if dense is not None else None)


def fluxbin_stream_probe(layer: PackedLayer, sink, stream=None) -> None:
    """Launch the measurement-only stream probe (the batch-1 kernel's weight requests without the table work) on
    ``sink``, a device buffer of at least 1024 bytes."""
    _check(lib().fluxbin_stream_probe(ctypes.byref(layer.layer), sink.data_ptr(), sink.numel() * sink.element_size(),
                                      _stream(stream)))


def fluxbin_rc_decompose(X, K: int, T: int, g: int, mask=None, prior=None, eps: float = 1e-12, stream=None):
    """RC_Decomp of X * mask (X: float32 [M, N] device tensor; mask: uint8 [N] device tensor or None) into K bases
    with one row scale per (row, block of g columns). prior: None, or (signs, alpha_r, alpha_c, gp) of earlier bases
    (as returned here) whose approximation is subtracted from X first. Returns (signs int32 [K, M, ceil(N/32)]
    canonical bit planes, alpha_r float64 [K, M, ceil(N/g)], alpha_c float64 [K, N])."""
    import torch
    M, N = X.shape
    ws_n = ctypes.c_size_t(0)
    _check(lib().fluxbin_rc_workspace_query(int(M), int(N), int(K), ctypes.byref(ws_n)))
    ws = torch.empty(ws_n.value, dtype=torch.uint8, device=X.device)
    signs = torch.empty(K, M, (N + 31) // 32, dtype=torch.int32, device=X.device)
    ar = torch.empty(K, M, -(-N // g), dtype=torch.float64, device=X.device)
    ac = torch.empty(K, N, dtype=torch.float64, device=X.device)
    ps, par, pac, gp = prior if prior is not None else (None, None, None, 1)
    kp = int(ps.shape[0]) if ps is not None else 0
    _check(lib().fluxbin_rc_decompose(X.data_ptr(), _ptr(mask), _ptr(ps), _ptr(par), _ptr(pac), kp, int(gp), int(M),
                                      int(N), int(K), int(T), int(g), float(eps), signs.data_ptr(), ar.data_ptr(),
                                      ac.data_ptr(), ws.data_ptr(), ws_n.value, _stream(stream)))
    return signs, ar, ac


def fluxbin_structural_search(W, hinv_diag, g: int, s: int, stream=None):
    """Column saliency with a diagonal inverse Hessian and the s most salient columns of every block of g columns.
    W: float32 [M, N] device tensor, hinv_diag: float64 [N] device tensor. Returns (scores float64 [N], indices int32,
    column mask uint8 [N])."""
    import torch
    M, N = W.shape
    n_sal = sum(min(s, N - b0) for b0 in range(0, N, g))
    scores = torch.empty(N, dtype=torch.float64, device=W.device)
    idx = torch.empty(n_sal, dtype=torch.int32, device=W.device)
    mask = torch.empty(N, dtype=torch.uint8, device=W.device)
    _check(lib().fluxbin_structural_search(W.data_ptr(), hinv_diag.data_ptr(), int(M), int(N), int(g), int(s),
                                           scores.data_ptr(), idx.data_ptr(), mask.data_ptr(), _stream(stream)))
    return scores, idx, mask



def fluxbin_get_tuning() -> Dict[str, int]:
    t = Tuning()
    _check(lib().fluxbin_get_tuning(ctypes.byref(t)))
    return {n: getattr(t, n) for n, _ in Tuning._fields_}


def fluxbin_set_tuning(values: Optional[Dict[str, int]]) -> None:
    """Set the process-wide launch-plan tuning (None: the library defaults)."""
    if values is None:
        _check(lib().fluxbin_set_tuning(None))
        return
    t = Tuning(**{n: int(values[n]) for n, _ in Tuning._fields_})
    _check(lib().fluxbin_set_tuning(ctypes.byref(t)))


class tuning:
    """Context manager: the current tuning with some fields overridden, restored on exit.
    Example: ``with fluxbin.tuning(mfma=0): ...`` runs the LUT batch kernel for every small batch."""

    def __init__(self, **overrides):
        self.overrides = overrides

    def __enter__(self):
        self.saved = fluxbin_get_tuning()
        new = dict(self.saved)
        for k, v in self.overrides.items():
            if k not in new:
                raise KeyError(f"unknown tuning field {k}")
            new[k] = int(v)
        fluxbin_set_tuning(new)
        return self

    def __exit__(self, *exc):
        fluxbin_set_tuning(self.saved)
        return False


def fluxbin_plan_query(layer: PackedLayer, B: int = 1) -> Dict[str, object]:
    """The launch plan a call with batch B would use (kernel name, workgroups, ...)."""
    p = PlanInfo()
    _check(lib().fluxbin_plan_query(ctypes.byref(layer.layer), int(B), ctypes.byref(p)))
    out = {n: getattr(p, n) for n, _ in PlanInfo._fields_}
    out["kernel_name"] = KERNEL_NAMES.get(p.kernel, str(p.kernel))
    return out
