"""The inputs built for the paper's ablations describe the same weights as the layer they come from (CPU)."""
import numpy as np
import pytest

import oracle
from synth import LayerSpec, make_activations, make_layer, vcm_off_equivalent


@pytest.mark.parametrize("spec", [
    LayerSpec("vcm_a", M=40, N=300, Kb=2, Ks=1, mu=8, S=17, g_r=128, g_s=17, outlier_frac=0.01, seed=9, layer_id=3),
    LayerSpec("vcm_b", M=33, N=256, Kb=3, Ks=2, mu=4, S=40, g_r=64, g_s=40, seed=10, layer_id=1),
    LayerSpec("vcm_none", M=20, N=128, Kb=2, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=11, layer_id=2),
], ids=lambda s: s.name)
def test_vcm_off_equivalent_same_result(spec):
    L = make_layer(spec)
    V = vcm_off_equivalent(L)
    assert V.spec.Ks == 0 and V.spec.S == 0 and V.spec.Kb == spec.Kb + (spec.Ks if spec.S else 0)
    x = make_activations(L, 2)
    assert np.array_equal(x, make_activations(V, 2))
    y, yv = oracle.gemv_dense(L, x), oracle.gemv_dense(V, x)
    assert np.max(np.abs(y - yv)) <= 1e-12 * np.max(np.abs(y))


def test_vcm_off_equivalent_needs_one_salient_row_scale():
    L = make_layer(LayerSpec("vcm_g", M=8, N=256, Kb=1, Ks=1, mu=8, S=40, g_r=128, g_s=16, seed=12))
    with pytest.raises(ValueError):
        vcm_off_equivalent(L)
