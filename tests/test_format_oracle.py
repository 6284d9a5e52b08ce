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
    assert fmt.chunk_info(s, 7) == ("pad", 0, 0, 6)      # a pad chunk uses the planes of the chunk before it
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
    assert vc["chunk_plane"].tolist() == [0, 1, 2, 3, 4, 5, 6, 6]


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


# ------------------------------------------------------------------------------------- fine row-scale groups (g < 128)

def test_fine_group_sizes_by_hand():
    # g_r = 64: two scales per global chunk and row; g_s = 8: sixteen per salient chunk (one per mu = 8 sub-vector).
    s = _layer(g_r=64, g_s=8, S=20).spec
    d = fmt.derived(s)
    assert (d["Gcg"], d["Gcs"], d["Gr"], d["Gs"]) == (2, 16, 5, 3)
    # 2 bases x 3 chunks = 6 global chunks (even: no separator), 1 salient chunk -> 7 chunks, 4 super-chunks
    assert (d["ngcp"], d["NC"], d["NSC"], d["nfc"]) == (6, 7, 4, 6)
    # planes: 6 global chunks x 2 + 1 salient chunk x 16
    assert (d["Pg"], d["NRP"]) == (12, 28)
    # three global bases: 9 global chunks (odd) and different layouts -> an inert separator chunk 9
    s3 = s.with_(Kb=3)
    d3 = fmt.derived(s3)
    assert (d3["ngcp"], d3["NC"], d3["nfc"]) == (10, 11, 10)
    assert fmt.chunk_info(s3, 9) == ("pad", 0, 0, fmt.chunk_info(s3, 8)[3])
    assert fmt.chunk_info(s3, 10) == ("s", 0, 0, d3["Pg"])
    # the same layout on both sides needs no separator
    assert fmt.derived(s3.with_(g_s=64, S=200))["ngcp"] == 9
    # coarse where the group covers the extent: g_s = 8 >= S = 5
    assert fmt.derived(s.with_(S=5, g_s=8))["Gcs"] == 1


def test_position_rotation_by_hand():
    # G = 2 groups of n = 8 positions (mu = 8): row 20 has floor(20/8) = 2 (group rotation 0) and 20 mod 8 = 4
    assert [fmt.position_subvector(q, 20, 16, 2) for q in range(16)] == \
        [4, 5, 6, 7, 0, 1, 2, 3, 12, 13, 14, 15, 8, 9, 10, 11]
    # row 9: group rotation 1, in-group rotation 1
    assert [fmt.position_subvector(q, 9, 16, 2) for q in range(16)] == \
        [9, 10, 11, 12, 13, 14, 15, 8, 1, 2, 3, 4, 5, 6, 7, 0]
    # G = 1 and G = 16 are the plain rotation (q + i) mod 16
    for G in (1, 16):
        assert [fmt.position_subvector(q, 5, 16, G) for q in range(16)] == [(q + 5) % 16 for q in range(16)]
    # any 16 consecutive rows read 16 different sub-vectors at every position (LDS banks)
    for G in (1, 2, 4, 8, 16):
        for q in range(16):
            assert sorted(fmt.position_subvector(q, i, 16, G) for i in range(16)) == list(range(16))
    for G in (1, 2, 4, 8, 16, 32):
        for q in range(32):
            assert sorted(fmt.position_subvector(q, i, 32, G) for i in range(32)) == list(range(32))


def test_single_bit_lands_where_the_definition_says_fine_mu8():
    L = _layer(M=40, g_r=64, g_s=8, S=20)
    L.signs[:] = 0
    L.sal_signs[:] = 0
    # row 20, global base 1, column 133 -> chunk 4, column 5 of the chunk: sub-vector 0 (group 0 of two), bit 5; chunk
    # 4 is in slot 1 for row 20. Position block b holds group (b + 2) mod 2 = b, position q = 8b + w holds sub-vector
    # 8b + (w + 4) mod 8: sub-vector 0 is at q = 4.
    i, j = 20, 133
    L.signs[1, i, j // 32] |= np.uint32(1 << (j % 32))
    dev = fmt.device_signs(L)
    assert np.argwhere(dev).tolist() == [[2, 1, 20, 4]]
    assert dev[2, 1, 20, 4] == 1 << 5


def test_fine_rscale_block_by_hand():
    L = _layer(M=40, g_r=64, g_s=8, S=20)
    s = L.spec
    rs = fmt.device_rscale(L)
    d = fmt.derived(s)
    assert rs.shape == (d["NRP"], 64)
    flat = rs.reshape(-1)
    # global base 1, chunk 2 of the base (columns 256..383: groups 4 and 5; group 5 does not exist, N = 300): block
    # (1*3 + 2)*2 = 10, rows of two scales. Row 20 (group rotation 0): slot 0 group 4, slot 1 group 5 (zero). Row 9
    # (rotation 1): slot 0 group 5 (zero), slot 1 group 4.
    blk = 10 * 64
    assert flat[blk + 20 * 2 + 0] == L.alpha_r[1, 20, 4] and flat[blk + 20 * 2 + 1] == 0
    assert flat[blk + 9 * 2 + 0] == 0 and flat[blk + 9 * 2 + 1] == L.alpha_r[1, 9, 4]
    # salient chunk (16 groups of 8 dense columns; S = 20 -> groups 0..2): block at plane Pg = 12, row 3 (group
    # rotation 3): slot b is group (b + 3) mod 16
    sblk = d["Pg"] * 64
    for b in range(16):
        grp = (b + 3) % 16
        want = L.alpha_sr[0, 3, grp] if grp < 3 else 0
        assert flat[sblk + 3 * 16 + b] == want
    assert np.all(rs.reshape(-1)[sblk + 40 * 16:sblk + 64 * 16] == 0)     # rows >= M


@pytest.mark.parametrize("mu,g_r,g_s,Kb", [(8, 64, 8, 3), (8, 32, 16, 2), (4, 64, 8, 3), (4, 16, 4, 1),
                                           (8, 128, 16, 3)])
def test_fine_layout_is_a_bijection(mu, g_r, g_s, Kb):
    L = _layer(mu=mu, M=70, g_r=g_r, g_s=g_s, S=40, Kb=Kb)
    rows = np.arange(fmt.derived(L.spec)["Mp"])
    dev = fmt.device_signs(L, rows)
    back = fmt.undo_device_signs(dev, L.spec, rows)
    assert np.array_equal(back, fmt.virtual_bits(L, rows))
    assert int(np.unpackbits(dev).sum()) == int(fmt.virtual_bits(L, rows).sum())
