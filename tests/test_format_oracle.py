"""Pins of the oracle's implementation of the packed device format: hand-worked examples, bijection and sizes."""
import numpy as np
import pytest

from oracle import format_oracle as fmt
from oracle import fluxbin_oracle as fo
from synth import LayerSpec, make_layer


def _layer(**kw):
    base = dict(M=40, N=300, Kb=2, Ks=1, mu=8, S=10, g_r=128, g_s=1000, seed=3)
    base.update(kw)
    return make_layer(LayerSpec("f", **base))


def test_derived_sizes_by_hand():
    L = _layer()
    d = fmt.derived(L.spec)
    # N = 300 -> 384 padded (3 chunks per global plane); S = 10 -> 128 (1 chunk); 2*3 + 1 = 7 chunks -> 4 super-chunks
    assert (d["Npad"], d["ncg"], d["Sv"], d["ncs"], d["NC"], d["NSC"], d["NCP"], d["V"]) == \
        (384, 3, 128, 1, 7, 4, 8, 1024)
    assert d["Mp"] == 64 and d["Gr"] == 3 and d["Gs"] == 1 and d["NRP"] == 7


def test_chunk_info_by_hand():
    s = _layer().spec
    assert fmt.chunk_info(s, 0) == ("g", 0, 0, 0)
    assert fmt.chunk_info(s, 2) == ("g", 0, 256, 2)
    assert fmt.chunk_info(s, 3) == ("g", 1, 0, 3)
    assert fmt.chunk_info(s, 6) == ("s", 0, 0, 6)
    assert fmt.chunk_info(s, 7) == ("pad", 0, 0, 0)
    s2 = s.with_(g_r=256)      # two chunks share a row-scale group
    assert [fmt.chunk_info(s2, c)[3] for c in range(7)] == [0, 0, 1, 2, 2, 3, 4]


def test_virtual_columns_by_hand():
    L = _layer()
    vc = fmt.virtual_columns(L)
    assert vc["xidx"][5] == 5 and vc["colscale"][5] == L.alpha_c[0, 5]
    assert vc["xidx"][299] == 299 and vc["xidx"][300] == 0xFFFF and vc["colscale"][300] == 0
    assert vc["xidx"][384 + 7] == 7 and vc["colscale"][384 + 7] == L.alpha_c[1, 7]
    t0 = 6 * 128
    assert vc["xidx"][t0 + 3] == L.sal_idx[3] and vc["colscale"][t0 + 3] == L.alpha_sc[0, L.sal_idx[3]]
    assert vc["xidx"][t0 + 10] == 0xFFFF
    assert np.all(vc["xidx"][7 * 128:] == 0xFFFF)
    assert vc["chunk_plane"].tolist() == [0, 1, 2, 3, 4, 5, 6, 0]


def test_single_bit_lands_where_the_definition_says_mu8():
    L = _layer(M=40)
    L.signs[:] = 0
    L.sal_signs[:] = 0
    # row 20 (upper half of a 32-row group), global base 1, column 133 -> chunk 4 (= 3 + 1), column 5 of the chunk:
    # sub-vector byte u = 0, bit 5. Chunk 4 is slot 0 of super-chunk 2 for lower-half rows, so for row 20 it is in
    # slot 1. Stored byte q holds u = (q + 20) mod 16, so u = 0 is at q = 12.
    i, j = 20, 133
    L.signs[1, i, j // 32] |= np.uint32(1 << (j % 32))
    dev = fmt.device_signs(L)
    nz = np.argwhere(dev)
    assert nz.tolist() == [[2, 1, 20, 12]]
    assert dev[2, 1, 20, 12] == 1 << 5


def test_single_bit_lands_where_the_definition_says_mu4():
    L = _layer(M=40, mu=4)
    L.signs[:] = 0
    L.sal_signs[:] = 0
    # row 3, global base 0, column 130 -> chunk 1, column 2 of the chunk: nibble u = 0, bit 2. Chunk 1 is slot 1 of
    # super-chunk 0. Stored nibble q holds u = (q + 3) mod 32, so u = 0 is at q = 29: byte 14, high nibble.
    L.signs[0, 3, 130 // 32] |= np.uint32(1 << (130 % 32))
    dev = fmt.device_signs(L)
    assert np.argwhere(dev).tolist() == [[0, 1, 3, 14]]
    assert dev[0, 1, 3, 14] == (1 << 2) << 4


def test_salient_bit_goes_to_the_dense_column():
    L = _layer(M=40)
    L.signs[:] = 0
    L.sal_signs[:] = 0
    t = 4
    j = int(L.sal_idx[t])
    L.sal_signs[0, 0, j // 32] |= np.uint32(1 << (j % 32))
    vb = fmt.virtual_bits(L, [0])
    assert np.argwhere(vb[0]).ravel().tolist() == [6 * 128 + t]


@pytest.mark.parametrize("mu", [4, 8])
def test_layout_is_a_bijection(mu):
    L = _layer(mu=mu, M=70)
    rows = np.arange(fmt.derived(L.spec)["Mp"])
    dev = fmt.device_signs(L, rows)
    back = fmt.undo_device_signs(dev, L.spec, rows)
    assert np.array_equal(back, fmt.virtual_bits(L, rows))
    # every stored bit count matches the virtual matrix (no bit duplicated or dropped)
    assert int(np.unpackbits(dev).sum()) == int(fmt.virtual_bits(L, rows).sum())


def test_virtual_bits_match_oracle_patterns():
    """The per-chunk sub-vector patterns of the virtual matrix equal the oracle's LUT indices."""
    L = _layer(M=8, N=256, S=20)
    p = fo.lut_indices(L)
    vb = fmt.virtual_bits(L, range(8)).reshape(8, -1, 128)
    sub = (vb.reshape(8, vb.shape[1], 16, 8).astype(np.int64) << np.arange(8)).sum(-1)
    for k in range(2):
        assert np.array_equal(sub[:, 2 * k:2 * k + 2].reshape(8, 32), p["global"][k])
    assert np.array_equal(sub[:, 4, :3], p["salient"][0])


def test_rscale_section():
    L = _layer(M=40, g_r=128)
    rs = fmt.device_rscale(L)
    assert rs.shape == (7, 64)
    assert np.array_equal(rs[4, :40], L.alpha_r[1, :, 1])
    assert np.array_equal(rs[6, :40], L.alpha_sr[0, :, 0])
    assert np.all(rs[:, 40:] == 0)


def test_packed_sizes_against_paper_storage_formula():
    """For the 7B attention shape the packed size is the paper's storage (App. C.2, with the salient count S and one
    salient row scale per row) plus this format's padding and per-virtual-column tables: within a few percent."""
    s = LayerSpec("a", M=4096, N=4096, Kb=2, Ks=1, mu=8, S=82, g_r=128, g_s=82)
    pb = fmt.packed_bytes(s)
    paper_bits = (s.Kb * (s.M * s.N + 16 * s.N + 16 * s.M * s.N / s.g_r)
                  + s.Ks * (s.M * s.S + 16 * s.S + 16 * s.M) + 16 * s.S)
    assert 1.0 <= pb["total"] / (paper_bits / 8) <= 1.03
    for k in ("signs", "rscale", "colscale", "xidx", "chunk_plane", "sal_idx"):
        assert pb["off_" + k] % 256 == 0
