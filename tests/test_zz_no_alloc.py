"""fluxbin_lut_gemv_noalloc (static device scratch, no allocation) against fluxbin_lut_gemv on the same layers.

The two entry points run the same launch plan and kernels, so their outputs must be bitwise equal; both are also
checked against the fp64 oracle (|y - y*| <= 2e-3 * max(|y*|, 1e-3 * max|y*|)). Two calls in a row, the second on a
smaller layer (fewer rows and columns, another launch plan), so the second call finds the first one's partial sums
in the shared scratch."""
import numpy as np
import pytest

import oracle
from synth import LayerSpec, make_activations, make_layer

from conftest import gpu_available
from gpu_util import log, pack_layer, x_tensor

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("no GPU")
    from paper_2608_15602_amd import fluxbin as fb
    fb.lib()


LARGE = LayerSpec("na_large", M=28672, N=8192, Kb=3, Ks=1, mu=8, S=410, g_r=128, g_s=410, outlier_frac=0.001,
                  seed=61)
SMALL = LayerSpec("na_small", M=6000, N=2048, Kb=2, Ks=1, mu=8, S=70, g_r=128, g_s=70, seed=62)
MU4 = LayerSpec("na_mu4", M=1500, N=777, Kb=3, Ks=2, mu=4, S=300, g_r=256, g_s=128, seed=63)


def _both(packed, xb, out_fp32):
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    x = x_tensor(xb)[0]
    dt = torch.float32 if out_fp32 else torch.float16
    y_ref = fb.fluxbin_lut_gemv(packed, x, out_fp32=out_fp32)
    y = torch.full((packed.shape.M,), float("nan"), dtype=dt, device="cuda")
    fb.fluxbin_lut_gemv_noalloc(packed, x, y, out_fp32=out_fp32)
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64), y_ref.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("out_fp32", [True, False])
def test_noalloc_equals_workspace_entry_point_two_calls(out_fp32):
    layers = []
    for spec in (LARGE, SMALL, MU4):
        L = make_layer(spec)
        layers.append((spec, L, pack_layer(L)))
    for spec, L, packed in layers:     # large first, then the smaller layers on the same scratch
        log(f"case noalloc {spec.name} M={spec.M} N={spec.N} mu={spec.mu} fp32={out_fp32}")
        xb = make_activations(L, 1)
        y, y_ref = _both(packed, xb, out_fp32)
        assert np.array_equal(y, y_ref), int(np.sum(y != y_ref))
        rows = np.unique(np.concatenate([np.arange(64), np.arange(spec.M - 64, spec.M),
                                         np.random.default_rng(1).choice(spec.M, 256, replace=False)]))
        r = oracle.parity_check(y[None, rows], oracle.gemv_dense(L, xb, rows=rows), rel=2e-3)
        log(f"  vs oracle: normwise={r['normwise']:.2e} ok={r['ok']}")
        assert r["ok"], r


def test_noalloc_rejects_layers_beyond_its_scratch():
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    spec = LayerSpec("na_tall", M=70000, N=128, Kb=1, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=64)
    log("case noalloc rejects M = 70000")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = x_tensor(make_activations(L, 1))[0]
    y = torch.zeros(spec.M, dtype=torch.float16, device="cuda")
    with pytest.raises(fb.FluxbinError) as e:
        fb.fluxbin_lut_gemv_noalloc(packed, x, y)
    assert e.value.status == fb.FLUXBIN_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert torch.count_nonzero(y).item() == 0
