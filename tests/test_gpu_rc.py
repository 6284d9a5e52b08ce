"""GPU parity of the weight decomposition (fluxbin_rc_decompose, fluxbin_structural_search, through the C ABI)
against the fp64 oracle (oracle/rc_oracle.py), and the decomposed layer through fluxbin_pack and the GEMV.

Bar: signs and selected columns bit-exact (both sides decide in fp64); row and column scales within 1e-9 relative
(fp64 sums in different orders), or within 1e-10 of the largest scale of the decomposition for the small scales of
later bases (their least-squares quotients divide residuals that cancel, which magnifies the fp64 rounding of the
residual relative to the scale itself); the GEMV of the decomposed layer within the hot path's 2e-3 rule."""
import numpy as np
import pytest

import oracle
from oracle import rc_oracle as rc
from synth import LayerSpec, make_weight_matrix
from synth.layers import SyntheticLayer

from conftest import gpu_available
from gpu_util import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("no GPU")
    from paper_2608_15602_amd import fluxbin as fb
    fb.lib()


def _bits(B):
    """int8 signs [K, M, N] -> canonical uint32 planes [K, M, ceil(N/32)] (bit set: +1)."""
    K, M, N = B.shape
    W = -(-N // 32)
    p = np.zeros((K, M, W * 32), dtype=np.uint8)
    p[:, :, :N] = (B == 1)
    return np.packbits(p, axis=-1, bitorder="little").view(np.uint32).reshape(K, M, W)


def _close(got, ref, what, rtol=1e-9):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    atol = 1e-10 * max(np.abs(ref).max(), 1e-300)
    err = np.abs(got - ref)
    bound = np.maximum(rtol * np.abs(ref), atol)
    worst = float((err / bound).max()) if ref.size else 0.0
    log(f"  {what}: max err / bound {worst:.2e}")
    assert np.all(err <= bound), what


def _gpu_rc(W, K, T, g, mask=None, prior=None):
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    X = torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).cuda()
    m = torch.from_numpy(mask.astype(np.uint8)).cuda() if mask is not None else None
    out = fb.fluxbin_rc_decompose(X, K, T, g, mask=m, prior=prior)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("K", [1, 2, 3])
def test_rc_decompose_matches_oracle(K):
    """Blocks of 64 columns with a ragged last block (N = 200), all columns."""
    W, _ = make_weight_matrix(96, 200, seed=30 + K)
    ref = rc.rc_decomp(W.astype(np.float64), np.ones(200, bool), K=K, T=4, g=64)
    signs, ar, ac = _gpu_rc(W, K, 4, 64)
    log(f"case rc K={K} M=96 N=200 g=64 T=4")
    assert np.array_equal(signs.cpu().numpy().view(np.uint32), _bits(ref["B"])), "signs differ"
    _close(ar.cpu().numpy(), ref["alpha_r"], "alpha_r")
    _close(ac.cpu().numpy(), ref["alpha_c"], "alpha_c")


def test_rc_decompose_masked_with_prior_matches_oracle():
    """The salient refinement of FluxBin-Hybrid: the residual of a 2-base global decomposition, decomposed on the
    salient column mask by two bases with one row scale per (row, block of g columns), as Alg. FluxBin-Hybrid does
    block by block."""
    import torch
    M, N, g = 128, 256, 64
    W, hinv = make_weight_matrix(M, N, seed=41, outlier_frac=0.02)
    ref = rc.hybrid_quantize(W.astype(np.float64), hinv, g=g, s=4, Kb=2, Ks=2, T=3)
    gs, gar, gac = _gpu_rc(W, 2, 3, g)
    from paper_2608_15602_amd import fluxbin as fb
    Wt = torch.from_numpy(W).cuda()
    scores, idx, mask = fb.fluxbin_structural_search(Wt, torch.from_numpy(hinv).cuda(), g, 4)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy().astype(np.int64), ref["sal_idx"]), "salient columns differ"
    _close(scores.cpu().numpy(), rc.saliency(W.astype(np.float64), hinv), "saliency", rtol=1e-12)
    ss, sar, sac = fb.fluxbin_rc_decompose(Wt, 2, 3, g, mask=mask, prior=(gs, gar, gac, g))
    torch.cuda.synchronize()
    assert np.array_equal(gs.cpu().numpy().view(np.uint32), _bits(ref["glob"]["B"])), "global signs differ"
    assert np.array_equal(ss.cpu().numpy().view(np.uint32), _bits(ref["sal"]["B"])), "salient signs differ"
    _close(sar.cpu().numpy(), ref["sal"]["alpha_r"], "alpha_sr")
    _close(sac.cpu().numpy(), ref["sal"]["alpha_c"], "alpha_sc")


def test_structural_search_matches_oracle():
    """Saliency scores and the per-block top-s columns, ragged last block."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    W, hinv = make_weight_matrix(300, 1000, seed=42, outlier_frac=0.01)
    for g, s in ((128, 8), (128, 16), (1000, 37), (7, 7)):
        scores, idx, mask = fb.fluxbin_structural_search(torch.from_numpy(W).cuda(), torch.from_numpy(hinv).cuda(), g, s)
        torch.cuda.synchronize()
        want = rc.structural_search(W.astype(np.float64), hinv, g, s)
        assert np.array_equal(idx.cpu().numpy().astype(np.int64), want), (g, s)
        m = np.zeros(1000, np.uint8)
        m[want] = 1
        assert np.array_equal(mask.cpu().numpy(), m), (g, s)


def test_decomposed_layer_through_pack_and_gemv():
    """A 2048 x 2048 weight matrix decomposed on the GPU in the paper's 2b-s8-g128 configuration (Alg. FluxBin-Hybrid:
    per 128-column block 8 salient columns, 2 global bases, 2 salient bases of the block's residual on them, one row
    scale per row and block on both branches), scales rounded to fp16, packed with one salient row scale per 8 dense
    columns (g_s = 8) and multiplied (B = 1 and 4) by the library: the result matches the GEMV oracle on the same
    layer; the signs match the decomposition oracle, and the hybrid error is below the global one."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    from gpu_util import pack_layer, run_gemm
    M, N, g, s, T = 2048, 2048, 128, 8, 4
    W, hinv = make_weight_matrix(M, N, seed=43, outlier_frac=0.01)
    Wt = torch.from_numpy(W).cuda()
    _, idx, mask = fb.fluxbin_structural_search(Wt, torch.from_numpy(hinv).cuda(), g, s)
    gs, gar, gac = fb.fluxbin_rc_decompose(Wt, 2, T, g)
    ss, sar, sac = fb.fluxbin_rc_decompose(Wt, 2, T, g, mask=mask, prior=(gs, gar, gac, g))
    torch.cuda.synchronize()
    ref = rc.hybrid_quantize(W.astype(np.float64), hinv, g=g, s=s, Kb=2, Ks=2, T=T)
    assert np.array_equal(gs.cpu().numpy().view(np.uint32), _bits(ref["glob"]["B"])), "global signs differ"
    assert np.array_equal(ss.cpu().numpy().view(np.uint32), _bits(ref["sal"]["B"])), "salient signs differ"
    sal = idx.cpu().numpy().astype(np.int32)
    S = len(sal)
    f16 = lambda a: np.ascontiguousarray(a.astype(np.float16)).view(np.uint16)
    assert S == s * (N // g)
    spec = LayerSpec("decomposed", M=M, N=N, Kb=2, Ks=2, mu=8, S=S, g_r=g, g_s=s, seed=0)
    L = SyntheticLayer(spec=spec, signs=gs.cpu().numpy().view(np.uint32), alpha_r=f16(gar.cpu().numpy()),
                       alpha_c=f16(gac.cpu().numpy()), sal_idx=sal, sal_signs=ss.cpu().numpy().view(np.uint32),
                       alpha_sr=f16(sar.cpu().numpy()), alpha_sc=f16(sac.cpu().numpy()),
                       outliers=np.zeros(0, np.int64))
    packed = pack_layer(L)
    rng = np.random.default_rng(44)
    for B in (1, 4):
        x = f16(rng.normal(size=(B, N)))
        y = run_gemm(packed, x)
        r = oracle.parity_check(y, oracle.gemv_dense(L, x))
        log(f"  decomposed layer B={B}: normwise {r['normwise']:.2e}")
        assert r["ok"], r
    Wg = rc.reconstruct(ref["glob"]["B"], ref["glob"]["alpha_r"], ref["glob"]["alpha_c"], g)
    Wh = Wg + rc.reconstruct(ref["sal"]["B"], ref["sal"]["alpha_r"], ref["sal"]["alpha_c"], g)
    assert ((W - Wh) ** 2).sum() < ((W - Wg) ** 2).sum()


@pytest.mark.parametrize("M,N,K,g,masked", [(1, 40, 2, 16, False), (33, 70, 4, 32, False), (50, 45, 3, 100, True),
                                            (300, 33, 1, 7, True)], ids=["one_row", "K4_ragged", "g_gt_N", "g7"])
def test_rc_decompose_edge_shapes(M, N, K, g, masked):
    """One row, N not a multiple of 32 (tail bits of the planes), four bases, a group wider than the matrix, a group of
    7 columns, masks; bit-exact signs and 1e-9 scales against the oracle."""
    W, _ = make_weight_matrix(M, N, seed=60 + M)
    mask = (np.random.default_rng(61).random(N) < 0.4) if masked else np.ones(N, bool)
    ref = rc.rc_decomp(W.astype(np.float64), mask, K=K, T=3, g=g)
    signs, ar, ac = _gpu_rc(W, K, 3, g, mask=mask if masked else None)
    log(f"case rc edge M={M} N={N} K={K} g={g} masked={masked}")
    assert np.array_equal(signs.cpu().numpy().view(np.uint32), _bits(ref["B"])), "signs differ"
    _close(ar.cpu().numpy(), ref["alpha_r"], "alpha_r")
    _close(ac.cpu().numpy(), ref["alpha_c"], "alpha_c")
