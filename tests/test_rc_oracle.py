"""Pins of the decomposition oracle (oracle/rc_oracle.py) against what the paper and the mathematics fix: exact
recovery of an exactly representable matrix, the least-squares scale updates (Prop. 3.2) against NumPy's lstsq, the
sign search (Prop. 3.3) against closed forms for K = 1 and K = 2, a non-increasing loss, the mask, and the saliency
selection against brute force over subsets."""
import itertools

import numpy as np

from oracle import rc_oracle as rc


def _rng(seed):
    return np.random.default_rng([seed, 7777])


def test_exactly_representable_matrix_is_recovered():
    """W = (r c^T) * S with one row scale per (row, block) and one column scale per column is reached exactly by one
    base (Def. RC decomposition): zero loss, the same signs, the same W."""
    rng = _rng(0)
    M, N, g = 24, 40, 8
    r = rng.uniform(0.5, 2.0, (M, N // g))
    c = rng.uniform(0.5, 2.0, N)
    S = np.where(rng.random((M, N)) < 0.5, 1, -1)
    W = np.repeat(r, g, axis=1) * c[None, :] * S
    out = rc.rc_decomp(W, np.ones(N, bool), K=1, T=40, g=g)
    assert np.array_equal(out["B"][0], S)
    What = rc.reconstruct(out["B"], out["alpha_r"], out["alpha_c"], g)
    assert np.abs(What - W).max() <= 1e-9 * np.abs(W).max()
    assert out["loss"][-1] <= 1e-16 * (W * W).sum()


def test_scale_updates_are_least_squares():
    """Prop. 3.2: each row (column) scale is the least-squares coefficient of the 1-column system (c_j B_ij) a = T_ij
    over the row (column), checked against numpy.linalg.lstsq."""
    rng = _rng(1)
    M, N = 9, 13
    T = rng.normal(size=(M, N))
    B = np.where(rng.random((M, N)) < 0.5, 1.0, -1.0)
    c = rng.uniform(0.2, 3.0, N)
    a = rc.row_update(T, B, c, eps=0.0)
    for i in range(M):
        ref = np.linalg.lstsq((c * B[i])[:, None], T[i], rcond=None)[0][0]
        assert abs(a[i] - ref) <= 1e-12 * max(1.0, abs(ref))
    r = rng.uniform(0.2, 3.0, (M, N))
    cc = rc.col_update(T, B, r, eps=0.0)
    for j in range(N):
        ref = np.linalg.lstsq((r[:, j] * B[:, j])[:, None], T[:, j], rcond=None)[0][0]
        assert abs(cc[j] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_sign_search_closed_forms():
    """Prop. 3.3 for K = 1: b = sign(x) (positive magnitudes). For K = 2 with m1 >= m2 >= 0 the four values
    +-m1 +- m2 are ordered, so the optimum is greedy: b1 = sign(x), b2 = sign(x - m1 b1)."""
    rng = _rng(2)
    x = rng.normal(size=(50, 60))
    m1 = rng.uniform(0.1, 2.0, x.shape)
    b = rc.sign_search(x, [m1])
    assert np.array_equal(b[0], np.where(x > 0, 1, -1))
    m2 = m1 * rng.uniform(0.0, 1.0, x.shape)
    b = rc.sign_search(x, [m1, m2])
    b1 = np.where(x > 0, 1, -1)
    b2 = np.where(x - m1 * b1 > 0, 1, -1)
    assert np.array_equal(b[0], b1) and np.array_equal(b[1], b2)


def test_sign_search_is_the_element_minimum():
    """Prop. 3.3 brute force for K = 3: no other combination is closer."""
    rng = _rng(3)
    x = rng.normal(size=(7, 11))
    mags = [rng.uniform(0.05, 1.5, x.shape) for _ in range(3)]
    b = rc.sign_search(x, mags)
    err = np.abs(x - sum(mags[k] * b[k] for k in range(3)))
    for combo in itertools.product((-1, 1), repeat=3):
        assert np.all(err <= np.abs(x - sum(mags[k] * combo[k] for k in range(3))) + 1e-15)


def test_loss_does_not_increase():
    """Every step of the alternating optimization solves its sub-problem exactly (Props. 3.2 and 3.3), so the loss
    after each round is at most the loss before it."""
    rng = _rng(4)
    W = rng.normal(size=(64, 96))
    W[:, 5] *= 20.0
    for K in (1, 2, 3):
        out = rc.rc_decomp(W, np.ones(96, bool), K=K, T=8, g=32)
        loss = out["loss"]
        assert np.all(loss[1:] <= loss[:-1] * (1 + 1e-12)), (K, loss)
        assert loss[-1] < (W * W).sum()


def test_mask_restricts_the_decomposition():
    """RC_Decomp with a column mask: signs are 0 and the reconstruction is exactly 0 off the mask, and the values of
    X off the mask are never used."""
    rng = _rng(5)
    W = rng.normal(size=(20, 30))
    mask = rng.random(30) < 0.3
    out = rc.rc_decomp(W, mask, K=2, T=4, g=30)
    assert np.all(out["B"][:, :, ~mask] == 0)
    What = rc.reconstruct(out["B"], out["alpha_r"], out["alpha_c"], 30)
    assert np.all(What[:, ~mask] == 0.0)
    W2 = W.copy()
    W2[:, ~mask] = rng.normal(size=(20, int((~mask).sum()))) * 100
    out2 = rc.rc_decomp(W2, mask, K=2, T=4, g=30)
    assert np.array_equal(out["B"], out2["B"]) and np.array_equal(out["alpha_r"], out2["alpha_r"])


def test_structural_search_is_the_best_subset_per_block():
    """Per block of g columns the chosen s columns maximize the total saliency S_j = sum_i W_ij^2 / hinv_jj^2 over
    every subset of size s (brute force)."""
    rng = _rng(6)
    M, N, g, s = 5, 14, 6, 2
    W = rng.normal(size=(M, N))
    hinv = rng.uniform(0.5, 2.0, N)
    S = (W * W).sum(axis=0) / hinv ** 2
    got = rc.structural_search(W, hinv, g, s)
    want = []
    for b0 in range(0, N, g):
        cols = list(range(b0, min(N, b0 + g)))
        best = max(itertools.combinations(cols, min(s, len(cols))), key=lambda sub: sum(S[j] for j in sub))
        want.extend(best)
    assert np.array_equal(got, np.array(sorted(want)))


def test_hybrid_refines_the_salient_columns():
    """FluxBin-Hybrid: the salient bases only touch the salient columns and lower the error there; elsewhere the
    hybrid approximation equals the global one."""
    rng = _rng(7)
    M, N, g = 48, 64, 16
    W = rng.normal(size=(M, N))
    W[:, [3, 40]] *= 15.0
    hinv = np.ones(N)
    h = rc.hybrid_quantize(W, hinv, g=g, s=2, Kb=2, Ks=1, T=5)
    Wg = rc.reconstruct(h["glob"]["B"], h["glob"]["alpha_r"], h["glob"]["alpha_c"], g)
    Ws = rc.reconstruct(h["sal"]["B"], h["sal"]["alpha_r"], h["sal"]["alpha_c"], g)
    sal = h["sal_idx"]
    assert 3 in sal and 40 in sal and len(sal) == 2 * (N // g)
    off = np.setdiff1d(np.arange(N), sal)
    assert np.all(Ws[:, off] == 0.0)
    err_g = ((W - Wg)[:, sal] ** 2).sum()
    err_h = ((W - Wg - Ws)[:, sal] ** 2).sum()
    assert err_h < 0.7 * err_g


def test_hybrid_salient_scales_are_per_block_closed_form():
    """Alg. FluxBin-Hybrid decomposes the salient residual block by block, so each salient base has one row scale per
    (row, block of g columns). With T = 0 rounds and one salient base the greedy initialization has a closed form: on
    the block's salient columns B_s = sign(R), the row scale is the mean |R| of the row over those columns (Prop. 3.2
    with unit column scales), and the column scale is sum_i a_i |R_ij| / sum_i a_i^2. Computed here directly from the
    global residual; a salient decomposition pooled over all blocks (one scale per row) gives other values."""
    rng = _rng(11)
    M, N, g, s = 6, 32, 8, 3
    W = rng.normal(size=(M, N))
    hinv = rng.uniform(0.5, 2.0, size=N)
    h = rc.hybrid_quantize(W, hinv, g=g, s=s, Kb=1, Ks=1, T=0)
    R = W - rc.reconstruct(h["glob"]["B"], h["glob"]["alpha_r"], h["glob"]["alpha_c"], g)
    sal = h["sal_idx"]
    assert h["sal"]["alpha_r"].shape == (1, M, N // g)
    for b in range(N // g):
        cols = [j for j in sal if b * g <= j < (b + 1) * g]
        assert len(cols) == s
        Rb = R[:, cols]
        a = np.abs(Rb).mean(axis=1)
        assert np.allclose(h["sal"]["alpha_r"][0, :, b], a, rtol=1e-10, atol=0)   # eps = 1e-12 in the quotients
        c = (a[:, None] * np.abs(Rb)).sum(axis=0) / (a * a).sum()
        assert np.allclose(h["sal"]["alpha_c"][0, cols], c, rtol=1e-10, atol=0)
        assert np.array_equal(h["sal"]["B"][0][:, cols], np.where(Rb >= 0, 1, -1))
    pooled = np.abs(R[:, sal]).mean(axis=1)
    assert not np.allclose(h["sal"]["alpha_r"][0, :, 0], pooled)


def test_hybrid_equals_its_blocks():
    """With a diagonal inverse Hessian the GPTQ compensation between blocks is zero, so the hybrid decomposition of W is
    the side-by-side concatenation of the hybrid decompositions of its column blocks (each a single block)."""
    rng = _rng(12)
    M, N, g, s = 20, 48, 16, 4
    W = rng.normal(size=(M, N))
    W[:, [5, 30]] *= 8.0
    hinv = rng.uniform(0.5, 2.0, size=N)
    h = rc.hybrid_quantize(W, hinv, g=g, s=s, Kb=2, Ks=2, T=3)
    for b in range(N // g):
        cols = slice(b * g, (b + 1) * g)
        hb = rc.hybrid_quantize(W[:, cols], hinv[cols], g=g, s=s, Kb=2, Ks=2, T=3)
        assert np.array_equal(hb["sal_idx"] + b * g, h["sal_idx"][b * s:(b + 1) * s])
        for br in ("glob", "sal"):
            assert np.array_equal(hb[br]["B"], h[br]["B"][:, :, cols])
            assert np.array_equal(hb[br]["alpha_r"][:, :, 0], h[br]["alpha_r"][:, :, b])
            assert np.array_equal(hb[br]["alpha_c"], h[br]["alpha_c"][:, cols])
    # and the same as RC_Decomp over all blocks at once (its row scales are per block too)
    glob = rc.rc_decomp(W, np.ones(N, bool), 2, 3, g)
    assert np.array_equal(glob["B"], h["glob"]["B"])
    assert np.allclose(glob["alpha_r"], h["glob"]["alpha_r"], rtol=1e-13, atol=0)
    mask = np.zeros(N, bool)
    mask[h["sal_idx"]] = True
    R = W - rc.reconstruct(glob["B"], glob["alpha_r"], glob["alpha_c"], g)
    salr = rc.rc_decomp(R, mask, 2, 3, g)
    assert np.array_equal(salr["B"], h["sal"]["B"])
    assert np.allclose(salr["alpha_r"], h["sal"]["alpha_r"], rtol=1e-10, atol=1e-14)
