"""Pins of the fp64 oracle to facts other than itself: printed paper values, closed forms, invariants, a textbook
special case and exact brute force on tiny inputs. CPU only."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import fluxbin_oracle as fo
from synth import LayerSpec, make_activations, make_layer


def _layer(M=24, N=40, Kb=2, Ks=1, mu=4, S=6, g_r=8, g_s=4, seed=7, **kw):
    return make_layer(LayerSpec("t", M=M, N=N, Kb=Kb, Ks=Ks, mu=mu, S=S, g_r=g_r, g_s=g_s, seed=seed, **kw))


# --------------------------------------------------------------------------- bit order and patterns

def test_sign_bits_hand_examples():
    w = np.array([[0x00000001, 0x00000000], [0x80000000, 0x00000002]], dtype=np.uint32)
    b = fo.sign_bits(w, 64)
    assert b[0].nonzero()[0].tolist() == [0]
    assert b[1].nonzero()[0].tolist() == [31, 33]
    pm = fo.sign_pm1(w[:1], 3)
    assert pm.tolist() == [[1.0, -1.0, -1.0]]


def test_sign_bits_against_shift_loop():
    rng = np.random.default_rng(3)
    w = rng.integers(0, 2**32, size=(5, 3), dtype=np.uint64).astype(np.uint32)
    b = fo.sign_bits(w, 96)
    for r in range(5):
        for j in range(96):
            assert b[r, j] == (int(w[r, j // 32]) >> (j % 32)) & 1


def test_patterns_hand_examples():
    bits = np.array([1, 0, 0, 0, 0, 0, 0, 1], dtype=np.uint8)
    assert fo.patterns(bits, 4).tolist() == [1, 8]
    assert fo.patterns(bits, 8).tolist() == [0x81]
    # a short tail run is padded with zero bits
    assert fo.patterns(np.array([0, 1, 1], dtype=np.uint8), 4).tolist() == [6]


# --------------------------------------------------------------------------- LUT-BSF closed forms (Eq. 14)

@pytest.mark.parametrize("mu", [4, 8])
def test_lut_closed_forms(mu):
    rng = np.random.default_rng(mu)
    x = rng.normal(size=mu)
    a = rng.lognormal(size=mu)
    lut = fo.lut_bsf(x[None], a[None])[0]
    xc = x * a
    full = (1 << mu) - 1
    assert lut.shape == (1 << mu,)
    assert np.isclose(lut[full], xc.sum(), rtol=1e-14, atol=1e-14)
    assert np.isclose(lut[0], -xc.sum(), rtol=1e-14, atol=1e-14)
    for n in range(mu):
        assert np.isclose(lut[1 << n], -xc.sum() + 2 * xc[n], rtol=1e-13, atol=1e-13)
    p = np.arange(1 << mu)
    assert np.allclose(lut[p] + lut[p ^ full], 0.0, atol=1e-13)


def test_lut_exact_enumeration():
    """Every entry equals an enumeration of signed sums in exact rationals (dyadic inputs keep fp64 exact)."""
    mu = 4
    xs = [Fraction(3, 4), Fraction(-5, 8), Fraction(1, 2), Fraction(7, 16)]
    al = [Fraction(2), Fraction(1, 4), Fraction(3, 2), Fraction(1)]
    lut = fo.lut_bsf(np.array([float(v) for v in xs])[None], np.array([float(v) for v in al])[None])[0]
    for p in range(16):
        want = Fraction(0)
        for n in range(mu):
            want += (xs[n] * al[n]) * (1 if (p >> n) & 1 else -1)
        assert Fraction(lut[p]) == want


# --------------------------------------------------------------------------- the product (Eqs. 10-15)

def _ones16(shape):
    return np.full(shape, 0x3C00, dtype=np.uint16)   # fp16 1.0


def test_textbook_integer_matvec():
    """Kb = 1, no salient base, unit scales and one row group: y = B x with B in {-1, +1}, checked against NumPy's
    integer matmul on integer activations."""
    L = _layer(M=33, N=48, Kb=1, Ks=0, S=0, mu=8, g_r=48, g_s=1)
    L.alpha_r[:] = _ones16(L.alpha_r.shape)
    L.alpha_c[:] = _ones16(L.alpha_c.shape)
    rng = np.random.default_rng(1)
    xi = rng.integers(-8, 9, size=(2, 48))
    x = xi.astype(np.float16).view(np.uint16)
    Bi = np.where(fo.sign_bits(L.signs[0], 48) == 1, 1, -1).astype(np.int64)
    want = (Bi @ xi.T).T
    assert np.array_equal(fo.gemv_dense(L, x), want.astype(np.float64))
    assert np.array_equal(fo.gemv_lut(L, x), want.astype(np.float64))


def _dyadic_layer(mu, N, S, g_r, g_s, Kb=2, Ks=1, M=6, seed=11):
    """A layer whose scales and activations are small dyadic numbers, so every fp64 step is exact."""
    L = _layer(M=M, N=N, Kb=Kb, Ks=Ks, S=S, mu=mu, g_r=g_r, g_s=g_s, seed=seed)
    rng = np.random.default_rng(seed)

    def dy(shape, lo, hi):
        return (rng.integers(lo, hi, size=shape) / 8.0).astype(np.float16).view(np.uint16)

    L.alpha_r[:] = dy(L.alpha_r.shape, 1, 16)
    L.alpha_c[:] = dy(L.alpha_c.shape, 1, 16)
    L.alpha_sr[:] = dy(L.alpha_sr.shape, 1, 16)
    L.alpha_sc[:] = dy(L.alpha_sc.shape, 1, 16)
    x = dy((2, N), -16, 17)
    return L, x


def _brute_force_fraction(L, x_bits):
    """Element-by-element evaluation of X W-hat^T in exact rationals, bits read with shifts from the canonical words,
    salient columns found by scanning the index list."""
    s = L.spec

    def F(u16):
        return Fraction(float(np.array(u16, dtype=np.uint16).view(np.float16)))

    def bit(words, i, j):
        return (int(words[i, j // 32]) >> (j % 32)) & 1

    B = x_bits.shape[0]
    out = [[Fraction(0)] * s.M for _ in range(B)]
    sal = [int(v) for v in L.sal_idx]
    for b in range(B):
        for i in range(s.M):
            acc = Fraction(0)
            for j in range(s.N):
                w = Fraction(0)
                for k in range(s.Kb):
                    sg = 1 if bit(L.signs[k], i, j) else -1
                    w += F(L.alpha_r[k, i, j // s.g_r]) * F(L.alpha_c[k, j]) * sg
                if j in sal:
                    t = sal.index(j)
                    for k in range(s.Ks):
                        sg = 1 if bit(L.sal_signs[k], i, j) else -1
                        w += F(L.alpha_sr[k, i, t // s.g_s]) * F(L.alpha_sc[k, j]) * sg
                acc += w * F(x_bits[b, j])
            out[b][i] = acc
    return out


@pytest.mark.parametrize("mu,N,S,g_r,g_s", [(4, 20, 5, 8, 4), (8, 24, 3, 8, 8), (4, 16, 0, 16, 1), (8, 19, 7, 16, 8)])
def test_exact_brute_force_tiny(mu, N, S, g_r, g_s):
    """Dense definition and LUT algorithm both equal the exact rational brute force on tiny inputs, including a
    column count that is not a multiple of mu (zero-padded tail sub-vector)."""
    L, x = _dyadic_layer(mu, N, S, g_r, g_s)
    want = _brute_force_fraction(L, x)
    yd = fo.gemv_dense(L, x)
    yl = fo.gemv_lut(L, x)
    for b in range(x.shape[0]):
        for i in range(L.spec.M):
            assert Fraction(yd[b, i]) == want[b][i]
            assert Fraction(yl[b, i]) == want[b][i]


@pytest.mark.parametrize("mu,g_r,g_s,S", [(4, 16, 8, 9), (8, 64, 16, 20), (8, 200, 1000, 13), (4, 200, 1000, 0)])
def test_dense_vs_lut_random(mu, g_r, g_s, S):
    L = _layer(M=70, N=200, Kb=3, Ks=2, S=S, mu=mu, g_r=g_r, g_s=g_s, seed=mu + S)
    x = make_activations(L, 3)
    yd = fo.gemv_dense(L, x)
    yl = fo.gemv_lut(L, x)
    assert np.max(np.abs(yd - yl)) <= 1e-12 * np.max(np.abs(yd))


def test_all_plus_one_closed_form():
    """All bits set: y_i = sum_k sum_grp alpha_r[i, grp] * (sum over the group of alpha_c[j] x_j), plus the same for
    the salient branch over its dense groups (scaled row sums)."""
    L = _layer(M=20, N=64, Kb=2, Ks=1, S=10, mu=8, g_r=16, g_s=8)
    L.signs[:] = 0xFFFFFFFF
    L.sal_signs[:] = 0xFFFFFFFF
    x = make_activations(L, 1)
    xf = fo.f16_to_f64(x)[0]
    s = L.spec
    want = np.zeros(s.M)
    for k in range(s.Kb):
        ax = fo.f16_to_f64(L.alpha_c[k]) * xf
        gsum = np.add.reduceat(ax, np.arange(0, s.N, s.g_r))
        want += fo.f16_to_f64(L.alpha_r[k]) @ gsum
    idx = L.sal_idx.astype(np.int64)
    for k in range(s.Ks):
        ax = (fo.f16_to_f64(L.alpha_sc[k]) * xf)[idx]
        gsum = np.add.reduceat(ax, np.arange(0, s.S, s.g_s))
        want += fo.f16_to_f64(L.alpha_sr[k]) @ gsum
    assert np.allclose(fo.gemv_dense(L, x)[0], want, rtol=1e-12, atol=1e-14)
    assert np.allclose(fo.gemv_lut(L, x)[0], want, rtol=1e-12, atol=1e-14)


def test_flip_whole_base_negates_its_contribution():
    L = _layer(M=30, N=64, Kb=3, Ks=1, S=6, mu=8, g_r=32, g_s=8)
    x = make_activations(L, 2)
    y = fo.gemv_dense(L, x)
    k = 1
    L0 = _layer(M=30, N=64, Kb=3, Ks=1, S=6, mu=8, g_r=32, g_s=8)
    L0.alpha_r[k] = 0
    y_without = fo.gemv_dense(L0, x)
    L.signs[k] = ~L.signs[k]          # all 64 columns are real columns (N = 64 fills both words)
    y_flip = fo.gemv_dense(L, x)
    assert np.allclose(y_flip, 2 * y_without - y, rtol=1e-12, atol=1e-12)
    assert np.allclose(fo.gemv_lut(L, x), y_flip, rtol=1e-12, atol=1e-12)


def test_flip_one_bit_changes_one_row_by_twice_the_term():
    L = _layer(M=12, N=64, Kb=2, Ks=0, S=0, mu=4, g_r=16, g_s=1)
    x = make_activations(L, 1)
    y = fo.gemv_lut(L, x)[0]
    k, i0, j0 = 1, 5, 37
    was = (int(L.signs[k, i0, j0 // 32]) >> (j0 % 32)) & 1
    L.signs[k, i0, j0 // 32] ^= np.uint32(1 << (j0 % 32))
    y2 = fo.gemv_lut(L, x)[0]
    term = fo.f16_to_f64(L.alpha_r[k, i0, j0 // 16]) * fo.f16_to_f64(L.alpha_c[k, j0]) * fo.f16_to_f64(x[0, j0])
    d = y2 - y
    assert np.allclose(np.delete(d, i0), 0.0, atol=1e-15)
    assert np.isclose(d[i0], (-2.0 if was else 2.0) * term, rtol=1e-10, atol=1e-15)


def test_vcm_equals_masked_full_width():
    """The VCM route (dense extraction + gather, Eqs. 12-13) equals the salient term of Eq. (10) written with the
    full-width mask (B_s * M) and per-column scales."""
    L = _layer(M=25, N=96, Kb=1, Ks=2, S=17, mu=4, g_r=96, g_s=8)
    L.alpha_r[:] = 0                      # isolate the salient branch
    x = make_activations(L, 2)
    xf = fo.f16_to_f64(x)
    s = L.spec
    mask = np.zeros(s.N)
    mask[L.sal_idx] = 1.0
    rank = np.full(s.N, -1)
    rank[L.sal_idx] = np.arange(s.S)
    want = np.zeros((2, s.M))
    for k in range(s.Ks):
        Bs = fo.sign_pm1(L.sal_signs[k], s.N) * mask[None, :]
        asr = np.zeros((s.M, s.N))
        for j in L.sal_idx:
            asr[:, j] = fo.f16_to_f64(L.alpha_sr[k, :, rank[j] // s.g_s])
        Wk = Bs * asr * fo.f16_to_f64(L.alpha_sc[k])[None, :]
        want += xf @ Wk.T
    assert np.allclose(fo.gemv_lut(L, x), want, rtol=1e-12, atol=1e-14)
    assert np.allclose(fo.gemv_dense(L, x), want, rtol=1e-12, atol=1e-14)


def test_salient_bits_off_the_set_are_ignored():
    L = _layer(M=16, N=64, S=5, mu=8, g_r=64, g_s=8)
    x = make_activations(L, 1)
    y = fo.gemv_lut(L, x)
    keep = np.zeros(64, dtype=bool)
    keep[L.sal_idx] = True
    bits = fo.sign_bits(L.sal_signs, 64)
    rnd = np.random.default_rng(0).integers(0, 2, size=bits.shape).astype(np.uint8)
    bits = np.where(keep[None, None, :], bits, rnd)
    L.sal_signs[:] = np.packbits(bits, axis=-1, bitorder="little").view("<u4")
    assert np.array_equal(fo.gemv_lut(L, x), y)
    assert np.allclose(fo.gemv_dense(L, x), y, rtol=1e-12, atol=1e-14)


def test_row_scale_group_indexing():
    """With activations nonzero only inside one row-scale group, y is linear in that group's row scale and does not
    depend on the others."""
    L = _layer(M=10, N=64, Kb=1, Ks=0, S=0, mu=8, g_r=16, g_s=1)
    x = np.zeros((1, 64), dtype=np.float16)
    x[0, 32:48] = np.random.default_rng(2).normal(size=16)
    xb = x.view(np.uint16)
    y = fo.gemv_lut(L, xb)
    L.alpha_r[0, :, [0, 1, 3]] = np.float16(7.0).view(np.uint16)
    assert np.array_equal(fo.gemv_lut(L, xb), y)
    ar = fo.f16_to_f64(L.alpha_r[0, :, 2])
    L.alpha_r[0, :, 2] = (ar * 2).astype(np.float16).view(np.uint16)
    assert np.allclose(fo.gemv_lut(L, xb), 2 * y, rtol=1e-12)
    assert np.allclose(fo.gemv_dense(L, xb), 2 * y, rtol=1e-12)


def test_power_of_two_scaling_is_exact():
    L = _layer(M=40, N=128, Kb=2, S=9, mu=8, g_r=64, g_s=16)
    x = make_activations(L, 2)
    x2 = (fo.f16_to_f64(x) * 2).astype(np.float16).view(np.uint16)
    assert np.array_equal(fo.gemv_dense(L, x2), 2 * fo.gemv_dense(L, x))


def test_lut_indices_match_bits():
    L = _layer(M=9, N=40, S=6, mu=4, g_r=8, g_s=4)
    p = fo.lut_indices(L)
    assert p["global"].shape == (2, 9, 10)
    assert p["salient"].shape == (1, 9, 2)
    for k in range(2):
        for i in range(9):
            for u in range(10):
                want = 0
                for n in range(4):
                    j = 4 * u + n
                    want |= ((int(L.signs[k, i, j // 32]) >> (j % 32)) & 1) << n
                assert p["global"][k, i, u] == want
    sal = [int(v) for v in L.sal_idx]
    for i in range(9):
        for u in range(2):
            want = 0
            for n in range(4):
                t = 4 * u + n
                if t < len(sal):
                    j = sal[t]
                    want |= ((int(L.sal_signs[0, i, j // 32]) >> (j % 32)) & 1) << n
            assert p["salient"][0, i, u] == want


# --------------------------------------------------------------------------- printed paper values

def _golden(name):
    with open(os.path.join(os.path.dirname(__file__), "golden", name)) as f:
        return json.load(f)


def test_abw_matches_paper_table():
    g = _golden("abw_groupsize.json")
    for row in g["rows"]:
        v = oracle.abw(g["M"], g["N"], g["Kb"], g["Ks"], row["g"], row["s"])
        assert abs(v - row["abw"]) <= g["tolerance"], (row, v)


def test_shared_memory_matches_paper_table():
    g = _golden("smem_mu_profile.json")
    for row in g["rows"]:
        b = oracle.smem_bytes(row["B_tile"], g["Kb"], g["K_tile"], row["mu"], g["M_tile"])
        assert b == row["kb"] * 1024, (row, b)


def test_effective_tflops_matches_paper_table():
    g = _golden("tile_dense_tflops.json")
    for M, N, _mt, _kt, lat2, tf2, lat4, tf4 in g["rows"]:
        assert abs(oracle.effective_tflops(M, N, 0, lat2 * 1e-6) - tf2) <= g["tolerance"]
        assert abs(oracle.effective_tflops(M, N, 0, lat4 * 1e-6) - tf4) <= g["tolerance"]


def test_effective_tflops_salient_term_matches_paper_table():
    """The N_sal term: the paper's hybrid-base TFLOPS (App. E.3) are reproduced with its salient columns counted
    (dropping the term misses most entries), at the salient width the table's figures follow (see the fixture)."""
    g = _golden("tile_saliency_tflops.json")
    miss = miss_without = total = 0
    for shape in g["shapes"]:
        M, N = shape["M"], shape["N"]
        for lat8, tf8, lat16, tf16 in shape["rows"]:
            for lat, tf in ((lat8, tf8), (lat16, tf16)):
                total += 1
                err = abs(oracle.effective_tflops(M, N, g["N_sal"], lat * 1e-6) - tf)
                assert err <= g["max_error"], (M, N, lat, tf, err)
                miss += err > g["tolerance"]
                miss_without += abs(oracle.effective_tflops(M, N, 0, lat * 1e-6) - tf) > g["tolerance"]
    assert total == 72 and miss <= g["max_mismatches"], miss
    assert miss_without > total // 2, miss_without


def test_effective_tflops_batch_factor():
    """Batch B (this library's small-batch figures; the paper defines the metric for one vector): B vectors in B
    times the latency are the batch-1 throughput, and B vectors in the batch-1 latency are B times it."""
    v1 = oracle.effective_tflops(4096, 4096, 128, 50e-6)
    assert np.isclose(oracle.effective_tflops(4096, 4096, 128, 8 * 50e-6, B=8), v1)
    assert np.isclose(oracle.effective_tflops(4096, 4096, 128, 50e-6, B=8), 8 * v1)


@pytest.mark.parametrize("mu,N,S,Kb,Ks", [(8, 256, 64, 2, 1), (4, 128, 24, 3, 2), (8, 512, 0, 1, 0)])
def test_complexity_counts_the_lut_algorithm(mu, N, S, Kb, Ks):
    """App. C.1's counts against the oracle's own LUT algorithm on a small layer: one table read per (base, row,
    sub-vector) the lookup path forms an index for, and 2^mu entries per (base, sub-vector) table."""
    M = 48
    spec = LayerSpec("cplx", M=M, N=N, Kb=Kb, Ks=Ks, mu=mu, S=S, g_r=N, g_s=max(S, 1), seed=9)
    L = make_layer(spec)
    idx = oracle.lut_indices(L)
    reads = idx["global"].size + idx["salient"].size
    tables = idx["global"].shape[0] * idx["global"].shape[2] + idx["salient"].shape[0] * idx["salient"].shape[2]
    c = oracle.complexity(M, N, S, Kb, Ks, mu)
    assert reads == c["read"], (reads, c)
    assert tables * 2 ** mu == c["build"], (tables, c)


def test_complexity_ratio():
    c = oracle.complexity(M=4096, N=4096, N_sal=256, Kb=2, Ks=2, mu=8)
    assert c["read"] / c["build"] == 4096 / 256
    dense = 4096 * 4096
    assert np.isclose(oracle.complexity(4096, 4096, 0, 2, 0, 8)["read"] / dense, 2 / 8)


# --------------------------------------------------------------------------- parity rule

def test_parity_rule():
    ref = np.array([[1.0, -2.0, 0.0, 1e-9, 3.0]])
    assert fo.parity_check(ref, ref)["ok"]
    y = ref.copy()
    y[0, 1] *= 1 + 1.9e-3
    assert fo.parity_check(y, ref)["ok"]
    y[0, 1] = ref[0, 1] * (1 + 2.1e-3)
    assert not fo.parity_check(y, ref)["ok"]
    y = ref.copy()
    y[0, 2] = 2e-3 * 1e-3 * 3.0 * 0.99      # inside the floored bound at a zero reference
    assert fo.parity_check(y, ref)["ok"]
    y[0, 2] = 2e-3 * 1e-3 * 3.0 * 1.01
    assert not fo.parity_check(y, ref)["ok"]
    y = ref.copy()
    y[0, 0] = np.nan
    assert not fo.parity_check(y, ref)["ok"]


# --------------------------------------------------------------------------- generator

def test_generator_is_deterministic():
    a = _layer(seed=5)
    b = _layer(seed=5)
    c = _layer(seed=6)
    assert np.array_equal(a.signs, b.signs) and np.array_equal(a.alpha_r, b.alpha_r)
    assert not np.array_equal(a.signs, c.signs)
    assert np.all(np.diff(a.sal_idx) > 0)
    xa = make_activations(a, 2)
    assert np.array_equal(xa, make_activations(b, 2))
    # tail bits past column N are zero
    t = _layer(N=40)
    assert np.all(t.signs[:, :, 1] >> 8 == 0)
