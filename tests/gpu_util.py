"""Shared helpers of the GPU tests: upload a synthetic layer, pack it through the C ABI, run the kernels."""
from __future__ import annotations

import sys

import numpy as np

from synth import make_activations, make_layer


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def upload(L, device="cuda"):
    import torch
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).view(dt)).to(device)
    w = dict(signs=t(L.signs, np.int32), alpha_r=t(L.alpha_r, np.int16), alpha_c=t(L.alpha_c, np.int16))
    if L.spec.S > 0:
        w["sal_idx"] = t(L.sal_idx.astype(np.int32), np.int32)
    if L.spec.S > 0 and L.spec.Ks > 0:
        w["sal_signs"] = t(L.sal_signs, np.int32)
        w["alpha_sr"] = t(L.alpha_sr, np.int16)
        w["alpha_sc"] = t(L.alpha_sc, np.int16)
    return w


def pack_layer(L, device="cuda"):
    from paper_2608_15602_amd import fluxbin as fb
    s = L.spec
    shape = fb.make_shape(s.M, s.N, s.Kb, s.Ks, s.mu, s.g_r, s.S, s.g_s)
    return fb.fluxbin_pack(shape, upload(L, device))


def x_tensor(x_bits, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x_bits).view(np.float16)).to(device)


def run_gemm(packed, x_bits, out_fp32=False, ws=None):
    """y [B, M] as float64 numpy, computed by the library (gemv for B = 1)."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    x = x_tensor(x_bits)
    if x.shape[0] == 1:
        y = fb.fluxbin_lut_gemv(packed, x[0], out_fp32=out_fp32, workspace=ws)[None]
    else:
        y = fb.fluxbin_lut_gemm_smallbatch(packed, x, out_fp32=out_fp32, workspace=ws)
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64)


def sample_rows(M: int, n: int = 768, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    rows = set(range(min(M, 64))) | set(range(max(0, M - 80), M))
    rows |= set(rng.choice(M, size=min(M, n), replace=False).tolist())
    return np.array(sorted(rows), dtype=np.int64)
