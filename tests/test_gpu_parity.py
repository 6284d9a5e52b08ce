"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bar: packing and LUT indices bit-exact; outputs within |y - y*| <= 2e-3 * max(|y*|, 1e-3 * max|y*| of the row)
(fp32 accumulation; x * alpha_c exact in fp32; fp16 output rounding 2^-11 relative). Full-size layers are checked on
sampled rows that the oracle computes one by one; the smaller ones on every row."""
import numpy as np
import pytest

import oracle
from oracle import format_oracle as fmt
from synth import CONFIGS, LayerSpec, config_layers, kernel_latency_layers, make_activations, make_layer, paper_config

from conftest import gpu_available
from gpu_util import log, pack_layer, run_gemm, sample_rows, x_tensor

pytestmark = pytest.mark.gpu

REL = 2e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("no GPU")
    from paper_2608_15602_amd import fluxbin as fb
    fb.lib()


def _check(y, y_ref, what):
    r = oracle.parity_check(y, y_ref, rel=REL)
    log(f"  {what}: normwise={r['normwise']:.2e} max_rel(>floor)={r['max_rel_above_floor']:.2e} "
        f"worst/bound={r['worst_bound_ratio']:.3f}")
    assert r["ok"], (what, r)


def _parity(spec, B, rows=None, out_fp32=False, packed=None, L=None):
    log(f"case {spec.name} M={spec.M} N={spec.N} Kb={spec.Kb} Ks={spec.Ks} mu={spec.mu} S={spec.S} g_r={spec.g_r} "
        f"g_s={spec.g_s} B={B} fp32={out_fp32}")
    L = L or make_layer(spec)
    packed = packed or pack_layer(L)
    x = make_activations(L, B)
    y = run_gemm(packed, x, out_fp32=out_fp32)
    if rows is None:
        y_ref = oracle.gemv_dense(L, x)
        _check(y, y_ref, "all rows")
    else:
        y_ref = oracle.gemv_dense(L, x, rows=rows)
        _check(y[:, rows], y_ref, f"{len(rows)} sampled rows")
    return L, packed, x, y


# ---------------------------------------------------------------------------------------------- packing, bit-exact

SMALL_SPECS = [
    LayerSpec("c1", M=512, N=256, Kb=2, Ks=1, mu=4, S=8, g_r=128, g_s=8, seed=0),
    LayerSpec("mu8_ragged", M=333, N=300, Kb=3, Ks=2, mu=8, S=77, g_r=128, g_s=77, seed=5),
    LayerSpec("mu4_ragged", M=100, N=200, Kb=1, Ks=1, mu=4, S=130, g_r=200, g_s=128, seed=6),
    LayerSpec("no_salient", M=64, N=128, Kb=2, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=7),
    # fine row-scale groups: g_r = 64 (two scales per global chunk), g_s = 8 (one per mu = 8 sub-vector), 9 global
    # chunks (odd: separator chunk); mu = 4 with g_r = 32 and g_s = 16; the paper's 2b-s16-g128
    LayerSpec("fine_mu8", M=333, N=300, Kb=3, Ks=2, mu=8, S=77, g_r=64, g_s=8, seed=8),
    LayerSpec("fine_mu4", M=100, N=200, Kb=1, Ks=1, mu=4, S=130, g_r=32, g_s=16, seed=9),
    LayerSpec("fine_s16", M=200, N=1024, Kb=2, Ks=2, mu=8, S=128, g_r=128, g_s=16, seed=10, sal_block=128),
]


@pytest.mark.parametrize("spec", SMALL_SPECS, ids=lambda s: s.name)
def test_pack_sections_bit_exact(spec):
    import torch
    log(f"case pack {spec.name}")
    L = make_layer(spec)
    packed = pack_layer(L)
    torch.cuda.synchronize()
    buf = packed.buf.cpu().numpy()
    pb = fmt.packed_bytes(spec)
    d = fmt.derived(spec)

    def sec(name, dtype, count):
        off = pb["off_" + name]
        return buf[off:off + count * np.dtype(dtype).itemsize].view(dtype)

    dev = fmt.device_signs(L)
    assert np.array_equal(sec("signs", np.uint8, dev.size), dev.reshape(-1))
    assert np.array_equal(sec("rscale", np.uint16, d["NRP"] * d["Mp"]), fmt.device_rscale(L).reshape(-1))
    vc = fmt.virtual_columns(L)
    assert np.array_equal(sec("colscale", np.uint16, d["V"]), vc["colscale"])
    assert np.array_equal(sec("xidx", np.uint16, d["V"]), vc["xidx"])
    assert np.array_equal(sec("chunk_plane", np.int32, d["NCP"]), vc["chunk_plane"])
    assert np.array_equal(sec("sal_idx", np.uint16, max(spec.S, 1)), fmt.device_sal_idx(L))
    hdr = buf[:8].view(np.uint32)
    assert hdr[0] == fmt.MAGIC and hdr[1] == fmt.VERSION


@pytest.mark.parametrize("spec", SMALL_SPECS, ids=lambda s: s.name)
def test_unpack_and_indices_bit_exact(spec):
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    log(f"case unpack/indices {spec.name}")
    L = make_layer(spec)
    packed = pack_layer(L)
    signs, dense = fb.fluxbin_unpack_canonical(packed)
    p = fb.fluxbin_debug_indices(packed)
    torch.cuda.synchronize()
    bits = oracle.sign_bits(L.signs, spec.N)
    got = oracle.sign_bits(signs.cpu().numpy().view(np.uint32), spec.N)
    assert np.array_equal(got, bits)
    if dense is not None:
        want = oracle.vcm_dense_bits(L)
        assert np.array_equal(oracle.sign_bits(dense.cpu().numpy().view(np.uint32), spec.S), want)
    # LUT indices of every (chunk, row, sub-vector) equal the oracle's patterns of the same columns
    idx = oracle.lut_indices(L)
    pc = p.cpu().numpy()
    per = 128 // spec.mu
    ncg = fmt.derived(spec)["ncg"]
    for k in range(spec.Kb):
        g = pc[k * ncg:(k + 1) * ncg].transpose(1, 0, 2).reshape(spec.M, -1)
        n = idx["global"].shape[2]
        assert np.array_equal(g[:, :n], idx["global"][k])
        assert np.all(g[:, n:] == 0)
    if spec.S > 0 and spec.Ks > 0:
        ncs = fmt.derived(spec)["ncs"]
        for k in range(spec.Ks):
            c0 = fmt.derived(spec)["ngcp"] + k * ncs   # after the separator chunk, if any
            sblk = pc[c0:c0 + ncs].transpose(1, 0, 2).reshape(spec.M, -1)
            n = idx["salient"].shape[2]
            assert np.array_equal(sblk[:, :n], idx["salient"][k])
    assert per * 2 * fmt.derived(spec)["NSC"] == pc.shape[0] * pc.shape[2]


def test_layer_survives_a_round_trip_through_its_header():
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    spec = SMALL_SPECS[1]
    log("case header round trip")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, 1)
    y1 = run_gemm(packed, x)
    copy = packed.buf.clone()
    again = fb.fluxbin_layer_from_header(packed.buf[:256].cpu().numpy().tobytes(), copy)
    y2 = run_gemm(again, x)
    assert np.array_equal(y1, y2)


# ---------------------------------------------------------------------------------------------- outputs

def test_config1_tiny_mu4():
    for spec in config_layers("c1_tiny", "128") + config_layers("c1_tiny", "N"):
        _parity(spec, 1)


@pytest.mark.parametrize("g_r", ["128", "N"])
def test_config2_attn7b(g_r):
    _parity(config_layers("c2_attn7b", g_r)[0], 1)


@pytest.mark.parametrize("g_r", ["128", "N"])
def test_config3_mlp7b(g_r):
    for spec in config_layers("c3_mlp7b", g_r):
        L = make_layer(spec)
        packed = pack_layer(L)
        for B in CONFIGS["c3_mlp7b"]["batches"]:
            _parity(spec, B, rows=sample_rows(spec.M, 512), packed=packed, L=L)


@pytest.mark.parametrize("g_r", ["128", "N"])
def test_config4_mlp70b(g_r):
    for spec in config_layers("c4_mlp70b", g_r):
        _parity(spec, 1, rows=sample_rows(spec.M, 768))


@pytest.mark.parametrize("g_r", ["128", "N"])
def test_config5_layer70b(g_r):
    import torch
    for spec in config_layers("c5_layer70b", g_r):
        L = make_layer(spec)
        packed = pack_layer(L)
        for B in CONFIGS["c5_layer70b"]["batches"]:
            _parity(spec, B, rows=sample_rows(spec.M, 128, seed=B), packed=packed, L=L)
        del packed
        torch.cuda.empty_cache()


def test_fused_decoder_layers_full_size():
    """The fused launches of the decoder layer (q|k|v as 10240 x 8192, gate|up as 57344 x 8192) at batch 1, 2, 4 and 16,
    sampled rows at full size, in the launch configuration the benchmark times."""
    import torch
    from synth import fused_decoder_layers
    for spec in fused_decoder_layers("128"):
        if not spec.name.endswith(("qkv", "gate_up")):
            continue
        L = make_layer(spec)
        packed = pack_layer(L)
        for B in (1, 2, 4, 16):
            _parity(spec, B, rows=sample_rows(spec.M, 128, seed=B), packed=packed, L=L)
        del packed
        torch.cuda.empty_cache()


def test_small_batch_kernel_choice_by_size():
    """The default small-batch kernel (mu = 8) moves from the matrix cores to the LUT batch kernel at 2.25 (B = 2) and
    3.5 (B = 3, 4) 1024-row units per CU, on a 256-CU device: 10240 x 8192 with 3 bases + 5% (980 units) takes the LUT
    batch kernel at B = 2..4 and the matrix cores at B = 8; 8192 x 8192 with 3 bases + 5% (784) the LUT batch kernel at
    B = 2 only; 8192 x 7168 (688) the LUT batch kernel at B = 2 and the row-complete matrix-core kernel at B = 3; the 7B
    gate/up layer (363) the matrix cores. Each choice also runs against the oracle on sampled rows."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    from synth import fused_decoder_layers, shard_layers
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("thresholds are stated for a 256-CU device")
    fused = {s.name: s for s in fused_decoder_layers("128")}
    c5 = {s.name: s for s in config_layers("c5_layer70b", "128")}
    down_p4 = [s for s in shard_layers(4, "128") if s.name == "down_p4"][0]
    gate_up7b = [s for s in config_layers("c3_mlp7b", "128") if s.name == "gate_up"][0]
    cases = [(fused["3b5pct_qkv"], {2: "lut_batch", 3: "lut_batch", 4: "lut_batch", 8: "mfma"}),
             (c5["3b5pct_q"], {2: "lut_batch", 3: "mfma", 4: "mfma"}),
             (down_p4, {2: "lut_batch", 3: "mfma_rows"}),
             (gate_up7b, {2: "mfma", 4: "mfma"})]
    for spec, want in cases:
        L = make_layer(spec)
        packed = pack_layer(L)
        for B, kernel in want.items():
            got = fb.fluxbin_plan_query(packed, B)["kernel_name"]
            log(f"plan {spec.name} {spec.M}x{spec.N} B={B}: {got}")
            assert got == kernel, (spec.name, B, got)
            _parity(spec, B, rows=sample_rows(spec.M, 64, seed=B), packed=packed, L=L)
        del packed
        torch.cuda.empty_cache()


@pytest.mark.parametrize("B", [1, 2, 4])
def test_24_unit_instances_full_size(B):
    """The fused 3 bases + 5% gate|up layer (57344 x 8192, 5488 units) on the instances that stage up to 24 units per
    1024-thread workgroup (batch-1 kernel at B = 1, LUT batch kernel at B = 2 and 4: one wave of 256 workgroups, the
    default) and with the 16 / 12-unit caps (two waves), sampled rows at full size, and determinism of the first."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    from synth import fused_decoder_layers
    spec = [s for s in fused_decoder_layers("128") if s.name == "3b5pct_gate_up"][0]
    L = make_layer(spec)
    packed = pack_layer(L)
    rows = sample_rows(spec.M, 256, seed=24 + B)
    x = make_activations(L, B)
    y_ref = oracle.gemv_dense(L, x, rows=rows)
    kernel = "batch1" if B == 1 else "lut_batch"
    for big, wgs in (("-1", 256), ("0", 512)):
        log(f"case 57344x8192 B={B}, big_units={big}")
        with fb.tuning(big_units=int(big)):
            info = fb.fluxbin_plan_query(packed, B)
            assert info["kernel_name"] == kernel and info["workgroups"] == wgs, info
            y = run_gemm(packed, x, out_fp32=True)
            if big == "-1":
                assert np.array_equal(run_gemm(packed, x, out_fp32=True), y), "repeat differs"
        _check(y[:, rows], y_ref, f"big_units={big}")
    del packed
    torch.cuda.empty_cache()


def test_kernel_variants_full_size():
    """The 28672 x 8192 layer in the kernel variants the benchmark times (mu 4, pure global bases, 2b + 1%), sampled
    rows at full size in the launch configuration the benchmark uses."""
    import torch
    from synth import kernel_variant_layers
    for spec in kernel_variant_layers("128"):
        _parity(spec, 1, rows=sample_rows(spec.M, 256, seed=5))
        torch.cuda.empty_cache()


@pytest.mark.parametrize("P", [2, 4, 8])
def test_shard_layers_full_size(P):
    """One rank's share of the 70B MLP layers at P ranks (up by output rows, down by input columns), sampled rows at
    full size in the launch configuration the benchmark uses, at batch 1 and 16."""
    import torch
    from synth import shard_layers
    for spec in shard_layers(P, "128"):
        L = make_layer(spec)
        packed = pack_layer(L)
        for B in (1, 16):
            _parity(spec, B, rows=sample_rows(spec.M, 256, seed=P), packed=packed, L=L)
        del packed
        torch.cuda.empty_cache()


def test_mu4_profile_layers_full_size():
    """The 7B attention and MLP layers at mu = 4 (the benchmark's mu profile), sampled rows at full size."""
    for cfg in ("c2_attn7b", "c3_mlp7b"):
        for spec in config_layers(cfg, "128"):
            _parity(spec.with_(mu=4, name=spec.name + "_mu4"), 1, rows=sample_rows(spec.M, 256, seed=7))


def test_vcm_off_equivalent_full_size():
    """The VCM ablation's layer (salient bases kept full width as extra global bases) gives the oracle's result of
    the original hybrid layer, on sampled rows of the 70B MLP up layer."""
    import torch
    from synth import vcm_off_equivalent
    spec = config_layers("c4_mlp70b", "128")[0]
    L = make_layer(spec)
    V = vcm_off_equivalent(L)
    packed = pack_layer(V)
    x = make_activations(L, 1)
    y = run_gemm(packed, x)
    rows = sample_rows(spec.M, 256, seed=6)
    _check(y[:, rows], oracle.gemv_dense(L, x, rows=rows), "VCM-off layer vs hybrid oracle")
    del packed
    torch.cuda.empty_cache()


EDGE_SPECS = [
    LayerSpec("one_row", M=1, N=128, Kb=1, Ks=1, mu=8, S=1, g_r=128, g_s=1, seed=11),
    LayerSpec("ragged_rows", M=1000, N=512, Kb=2, Ks=1, mu=8, S=33, g_r=256, g_s=33, seed=12),
    LayerSpec("ragged_cols", M=300, N=300, Kb=2, Ks=1, mu=8, S=5, g_r=128, g_s=5, seed=13),
    LayerSpec("all_salient", M=256, N=256, Kb=1, Ks=1, mu=8, S=256, g_r=256, g_s=128, seed=14),
    LayerSpec("salient_groups", M=640, N=1024, Kb=2, Ks=2, mu=8, S=300, g_r=512, g_s=128, seed=15),
    LayerSpec("four_bases", M=513, N=1024, Kb=4, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=16),
    LayerSpec("mu4_ragged", M=777, N=260, Kb=2, Ks=1, mu=4, S=20, g_r=260, g_s=20, seed=17),
    LayerSpec("tiny_N", M=70, N=7, Kb=2, Ks=1, mu=4, S=3, g_r=7, g_s=3, seed=18),
    LayerSpec("one_col", M=100, N=1, Kb=2, Ks=1, mu=8, S=1, g_r=1, g_s=1, seed=25),
    LayerSpec("one_by_one", M=1, N=1, Kb=1, Ks=0, mu=8, S=0, g_r=1, g_s=1, seed=26),
    # fine row-scale groups (group shorter than a 128-column chunk) on the global side, the salient side or both
    LayerSpec("fine_g64_s8", M=1000, N=300, Kb=3, Ks=2, mu=8, S=77, g_r=64, g_s=8, seed=19),
    LayerSpec("fine_g8_s16", M=700, N=512, Kb=2, Ks=1, mu=8, S=100, g_r=8, g_s=16, seed=20),
    LayerSpec("fine_g32_s64", M=300, N=1024, Kb=1, Ks=1, mu=8, S=300, g_r=32, g_s=64, seed=21),
    LayerSpec("fine_global_only", M=600, N=384, Kb=2, Ks=0, mu=8, S=0, g_r=16, g_s=1, seed=22),
    LayerSpec("fine_one_row", M=1, N=128, Kb=1, Ks=1, mu=8, S=16, g_r=64, g_s=8, seed=23),
    LayerSpec("fine_mu4", M=333, N=260, Kb=2, Ks=1, mu=4, S=40, g_r=16, g_s=4, seed=24),
]


@pytest.mark.parametrize("spec", EDGE_SPECS, ids=lambda s: s.name)
@pytest.mark.parametrize("B", [1, 3, 9])
def test_edge_shapes(spec, B):
    """B = 1: batch-1 kernels (the plan's choice, and the split-tile kernel with the row-complete one switched off);
    B = 3: LUT batch kernel (mu = 8) or matrix cores (mu = 4); B = 9: matrix cores."""
    _parity(spec, B)
    if B == 1:
        _with_env({"FLUXBIN_ROWS": "0"}, lambda: _parity(spec, B))


@pytest.mark.parametrize("spec", kernel_latency_layers(), ids=lambda s: s.name)
def test_paper_kernel_latency_configs_full_size(spec):
    """The operator shapes and configurations of the paper's kernel-latency table (App. E.4): 2b-g128, 2b-s8-g128
    (structured selection of 8 salient columns per 128, one salient row scale per row and block, Ks = Kb = 2),
    2b-s16-g128 and 4b-g128 at full size in the benchmark's launch configuration, sampled rows against the oracle."""
    rows = sample_rows(spec.M, 384, seed=spec.layer_id)
    _parity(spec, 1, rows=rows)


ROWS_SPECS = [
    LayerSpec("rows_mu8_ragged", M=333, N=300, Kb=3, Ks=2, mu=8, S=77, g_r=128, g_s=77, seed=60),
    LayerSpec("rows_mu4_ragged", M=100, N=201, Kb=1, Ks=1, mu=4, S=130, g_r=201, g_s=128, seed=61),
    LayerSpec("rows_no_salient", M=64, N=128, Kb=2, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=62),
    LayerSpec("rows_mu8_wide", M=1000, N=5000, Kb=2, Ks=1, mu=8, S=100, g_r=5000, g_s=100, seed=63),
    LayerSpec("rows_mu4_many", M=257, N=16384, Kb=1, Ks=1, mu=4, S=128, g_r=128, g_s=128, seed=64),
    # the paper's s8 / s16 configurations (16 / 8 fine row-scale groups per salient chunk), ragged M and N
    paper_config("rows_2b-s8", 333, 1000, 2, 8, 128, seed=66),
    paper_config("rows_2b-s16", 200, 2048, 2, 16, 128, seed=67),
    paper_config("rows_3b-s8_separator", 300, 1100, 3, 8, 128, seed=68),   # 27 global chunks: an inert separator
]


@pytest.mark.parametrize("nt,depth", [(1024, 2), (512, 4), (256, 6)])
def test_rows_kernel_instances(nt, depth):
    """Every workgroup size (4, 8, 16 wavefronts) and request depth of the row-complete kernel: both packed mu and both
    fine salient group counts."""
    specs = [LayerSpec(f"rows_inst_mu{mu}", M=500, N=1500, Kb=2, Ks=1, mu=mu, S=60, g_r=128, g_s=60, seed=65)
             for mu in (8, 4)]
    specs += [paper_config(f"rows_inst_s{sv}", 500, 1500, 2, sv, 128, seed=66) for sv in (8, 16)]
    for spec in specs:
        _with_env({"FLUXBIN_ROWS": "1", "FLUXBIN_NT": str(nt), "FLUXBIN_DEPTH": str(depth)},
                  lambda: _parity(spec, 1, out_fp32=True))


@pytest.mark.parametrize("spec", ROWS_SPECS, ids=lambda s: s.name)
def test_rows_kernel_matches_oracle(spec):
    """The row-complete batch-1 kernel (forced) on every row: both packed mu, ragged M and N, salient chunks, no
    salient part, the widest N its activation staging takes, and more super-chunks than four wavefronts hold (its
    512-thread instance); and it is the kernel the plan reports."""
    from paper_2608_15602_amd import fluxbin as fb
    L = make_layer(spec)
    packed = pack_layer(L)
    with fb.tuning(rows=1):
        assert fb.fluxbin_plan_query(packed, 1)["kernel_name"] == "rows"
        _, _, x, y = _parity(spec, 1, out_fp32=True, packed=packed, L=L)
        assert np.array_equal(run_gemm(packed, x, out_fp32=True), y), "repeat differs"
    y16 = _with_env({"FLUXBIN_ROWS": "1"}, lambda: run_gemm(packed, x))
    _check(y16, oracle.gemv_dense(L, x), "fp16 output")


@pytest.mark.parametrize("spec", kernel_latency_layers() + config_layers("c3_mlp7b", "128"), ids=lambda s: s.name)
def test_rows_kernel_full_size(spec):
    """The row-complete kernel (forced where the layer allows it) on the App. E.4 shapes (2b, s8, s16, 4b) and the 7B
    MLP layers at full size, sampled rows against the oracle."""
    _with_env({"FLUXBIN_ROWS": "1"}, lambda: _parity(spec, 1, rows=sample_rows(spec.M, 256, seed=spec.M)))


ROWS32_SPECS = [s for s in ROWS_SPECS if s.mu == 8] + [
    LayerSpec("rows32_one_row", M=1, N=256, Kb=2, Ks=1, mu=8, S=20, g_r=128, g_s=20, seed=69),
    LayerSpec("rows32_17_rows", M=17, N=640, Kb=1, Ks=1, mu=8, S=200, g_r=640, g_s=200, seed=70),
    LayerSpec("rows32_ragged_47", M=47, N=1300, Kb=3, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=71),
    # fine salient groups on rows 16 and 32 apart (same stored byte order), M across and past 48-row workgroups
    paper_config("rows32_2b-s16_ragged_101", 101, 700, 2, 16, 128, seed=73),
    paper_config("rows32_3b-s8_ragged_50", 50, 2304, 3, 8, 128, seed=74),
]


@pytest.mark.parametrize("rb", [2, 3])
@pytest.mark.parametrize("spec", ROWS32_SPECS, ids=lambda s: s.name)
def test_rows_kernel_32_rows_matches_oracle(spec, rb):
    """The row-complete kernel's 32- and 48-row workgroups (two or three rows per lane, forced) on every row: ragged M
    below, across and above them (48-row workgroups past the padded rows), salient chunks or none, coarse or 8 / 16
    fine salient row-scale groups, wide N; deterministic, the plan reports it; and a mu = 4 layer, which it does not
    take, keeps another kernel."""
    from paper_2608_15602_amd import fluxbin as fb
    L = make_layer(spec)
    packed = pack_layer(L)
    with fb.tuning(rows=rb):
        info = fb.fluxbin_plan_query(packed, 1)
        assert info["kernel_name"] == "rows" and info["rows_per_tile"] == 16 * rb, info
        _, _, x, y = _parity(spec, 1, out_fp32=True, packed=packed, L=L)
        assert np.array_equal(run_gemm(packed, x, out_fp32=True), y), "repeat differs"
    other = LayerSpec("rows32_mu4", M=100, N=300, Kb=1, Ks=1, mu=4, S=20, g_r=128, g_s=20, seed=72)
    with fb.tuning(rows=rb):
        assert fb.fluxbin_plan_query(pack_layer(make_layer(other)), 1)["kernel_name"] != "rows"


@pytest.mark.parametrize("spec", kernel_latency_layers() + config_layers("c3_mlp7b", "128"), ids=lambda s: s.name)
@pytest.mark.parametrize("rb", [2, 3])
def test_rows_kernel_32_rows_full_size(spec, rb):
    """The 32- and 48-row workgroups of the row-complete kernel (forced) on the App. E.4 shapes (2b, s8, s16, 4b) and
    the 7B MLP layers at full size, sampled rows (the last ones included) against the oracle."""
    _with_env({"FLUXBIN_ROWS": str(rb)}, lambda: _parity(spec, 1, rows=sample_rows(spec.M, 256, seed=spec.M + rb)))


@pytest.mark.parametrize("B", [2, 4, 8])
@pytest.mark.parametrize("spec", [paper_config("2b-s8-g128_small", 1536, 2048, 2, 8, 128),
                                  paper_config("3b-s16-g128_ragged", 1000, 1100, 3, 16, 128, seed=9)],
                         ids=lambda s: s.name)
def test_paper_config_small_batch(spec, B):
    """Paper-configuration layers (8 or 16 fine salient row-scale groups per chunk) at B <= 8: B launches of the batch-1
    kernels (the plan reports one-row batch tiles), every row against the oracle, and within tolerance of the generic
    kernel that 16-row tiles run (FLUXBIN_BATCH_TILE=16)."""
    from paper_2608_15602_amd import fluxbin as fb
    L = make_layer(spec)
    packed = pack_layer(L)
    info = fb.fluxbin_plan_query(packed, B)
    assert (info["batch_tile_rows"], info["batch_tiles"]) == (1, B), info
    assert info["kernel_name"] in ("batch1", "rows"), info
    _, _, x, y = _parity(spec, B, out_fp32=True, packed=packed, L=L)
    env = {"FLUXBIN_BATCH_TILE": "16"}
    assert _with_env(env, lambda: fb.fluxbin_plan_query(packed, B))["kernel_name"] == "generic"
    _check(y, _with_env(env, lambda: run_gemm(packed, x, out_fp32=True)), "per-row batch-1 launches vs generic kernel")


def test_paper_config_small_batch_full_size():
    """The App. E.4 5120 x 13824 s8 and s16 layers at B = 3 (three batch-1 launches), sampled rows at full size."""
    for spec in kernel_latency_layers():
        if spec.M == 5120 and spec.N == 13824 and "-s" in spec.name:
            _parity(spec, 3, rows=sample_rows(spec.M, 128, seed=3))


@pytest.mark.parametrize("spec", [
    LayerSpec("mu4_b1_a", M=3000, N=2048, Kb=2, Ks=1, mu=4, S=70, g_r=128, g_s=70, seed=51),
    LayerSpec("mu4_b1_b", M=1500, N=777, Kb=3, Ks=2, mu=4, S=300, g_r=256, g_s=128, seed=52),
    LayerSpec("mu4_b1_c", M=64, N=300, Kb=1, Ks=0, mu=4, S=0, g_r=300, g_s=1, seed=53),
], ids=lambda s: s.name)
def test_mu4_batch1_kernel_matches_oracle_and_generic(spec):
    """mu = 4 at batch 1: the split-tile batch-1 kernel (16-entry tables) matches the oracle on every row, and the
    generic and row-complete kernels' results within the tolerance."""
    L, packed, x, y = _with_env({"FLUXBIN_ROWS": "0"}, lambda: _parity(spec, 1, out_fp32=True))
    y_gen = _with_env({"FLUXBIN_GENERIC": "1"}, lambda: run_gemm(packed, x, out_fp32=True))
    _check(y, y_gen, "batch-1 kernel vs generic kernel")
    y_rows = _with_env({"FLUXBIN_ROWS": "1"}, lambda: run_gemm(packed, x, out_fp32=True))
    _check(y, y_rows, "batch-1 kernel vs row-complete kernel")


def test_fp32_output_and_generic_kernel_at_batch1():
    spec = LayerSpec("gen", M=2000, N=1024, Kb=2, Ks=1, mu=8, S=40, g_r=128, g_s=40, seed=21)
    L, packed, x, y = _parity(spec, 1, out_fp32=True)
    y2 = _with_env({"FLUXBIN_GENERIC": "1"}, lambda: run_gemm(packed, x, out_fp32=True))
    _check(y2, oracle.gemv_dense(L, x), "generic kernel at batch 1")


# Small-batch kernels: the split-tile matrix-core kernel (FLUXBIN_MFMA=1, FLUXBIN_MFMA_ROWS=0; the default for mu = 4
# and for B > 4 on larger layers), the row-complete matrix-core kernel (FLUXBIN_MFMA_ROWS=1: B = 2..8 where it fits;
# the default on layers with few rows), the mu = 8 LUT batch kernel (FLUXBIN_MFMA=0; the default for mu = 8 up to B = 4
# on large layers) and the generic LUT kernel (FLUXBIN_GENERIC=1; with FLUXBIN_MFMA=0 also the mu = 4 small-batch path).
SMALL_BATCH_KERNELS = {"mfma": {"FLUXBIN_MFMA": "1", "FLUXBIN_MFMA_ROWS": "0"}, "mfma_rows": {"FLUXBIN_MFMA_ROWS": "1"},
                       "lut_batch": {"FLUXBIN_MFMA": "0"},
                       "generic": {"FLUXBIN_GENERIC": "1"}}


def _with_env(env, fn):
    """Run fn with launch-plan tuning fields overridden (named like their FLUXBIN_* environment variables), restored
    afterwards (fluxbin_set_tuning: the library reads the environment only once per process)."""
    from paper_2608_15602_amd import fluxbin as fb
    kw = {k[len("FLUXBIN_"):].lower(): int(v) for k, v in env.items()}
    with fb.tuning(**kw):
        return fn()


@pytest.mark.parametrize("kernel", list(SMALL_BATCH_KERNELS))
@pytest.mark.parametrize("mu", [8, 4])
@pytest.mark.parametrize("B", [2, 5, 9, 12, 16])
def test_batch_rows_equal_batch1(B, mu, kernel):
    """Each batch row of every small-batch kernel matches the oracle (rows of several split tiles, a ragged last
    tile, B not a multiple of four)."""
    spec = LayerSpec("bat", M=1536, N=2048, Kb=2, Ks=1, mu=mu, S=61, g_r=128, g_s=61, seed=22)
    _with_env(SMALL_BATCH_KERNELS[kernel], lambda: _parity(spec, B, out_fp32=True))


MR_SPECS = [
    LayerSpec("mr_mu8", M=1000, N=1000, Kb=2, Ks=1, mu=8, S=40, g_r=128, g_s=40, seed=81),
    LayerSpec("mr_mu4", M=700, N=2048, Kb=3, Ks=1, mu=4, S=33, g_r=128, g_s=33, seed=82),
    LayerSpec("mr_1base_32rows", M=4100, N=640, Kb=1, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=83),
    LayerSpec("mr_mu4_32rows", M=5000, N=700, Kb=2, Ks=1, mu=4, S=20, g_r=128, g_s=20, seed=84),
]


@pytest.mark.parametrize("B", [2, 3, 5, 8])
@pytest.mark.parametrize("spec", MR_SPECS, ids=lambda s: s.name)
def test_mfma_rows_kernel_matches_oracle(spec, B):
    """The row-complete matrix-core kernel (16 or 32 rows per workgroup, every super-chunk of them): every row and
    batch row against the oracle on ragged layers (M and N not multiples of the tiles, one and three bases, salient
    columns or none, mu 8 and 4), bitwise repeatable, and within tolerance of the split-tile matrix-core kernel."""
    from paper_2608_15602_amd import fluxbin as fb
    L = make_layer(spec)
    packed = pack_layer(L)
    env = SMALL_BATCH_KERNELS["mfma_rows"]
    info = _with_env(env, lambda: fb.fluxbin_plan_query(packed, B))
    assert info["kernel_name"] == "mfma_rows", info
    assert info["rows_per_tile"] == (16 if -(-spec.M // 16) <= 256 else 32), info
    _, _, x, y = _with_env(env, lambda: _parity(spec, B, packed=packed, L=L, out_fp32=True))
    assert np.array_equal(_with_env(env, lambda: run_gemm(packed, x, out_fp32=True)), y), "repeat differs"
    y_split = _with_env(SMALL_BATCH_KERNELS["mfma"], lambda: run_gemm(packed, x, out_fp32=True))
    _check(y, y_split, "row-complete vs split-tile matrix-core kernel")


MR_EDGE_SPECS = [
    LayerSpec("mr_one_row_one_col", M=1, N=1, Kb=1, Ks=0, mu=8, S=0, g_r=1, g_s=1, seed=85),
    LayerSpec("mr_17x129_mu4", M=17, N=129, Kb=2, Ks=1, mu=4, S=3, g_r=128, g_s=3, seed=86),
    LayerSpec("mr_33x300_salient_only_chunk", M=33, N=300, Kb=1, Ks=2, mu=8, S=130, g_r=128, g_s=130, seed=87),
]


@pytest.mark.parametrize("B", [2, 7])
@pytest.mark.parametrize("spec", MR_EDGE_SPECS, ids=lambda s: s.name)
def test_mfma_rows_kernel_edge_shapes(spec, B):
    """Degenerate shapes on the row-complete matrix-core kernel (one row and one column; fewer super-chunks than
    wavefronts; a ragged mu = 4 layer; two salient bases over more than one salient chunk) and on a 32-row matrix-core
    launch of the same layers: every row against the oracle."""
    from paper_2608_15602_amd import fluxbin as fb
    L = make_layer(spec)
    packed = pack_layer(L)
    env = SMALL_BATCH_KERNELS["mfma_rows"]
    assert _with_env(env, lambda: fb.fluxbin_plan_query(packed, B))["kernel_name"] == "mfma_rows"
    _with_env(env, lambda: _parity(spec, B, packed=packed, L=L, out_fp32=True))
    _parity(spec, 16 + B, packed=packed, L=L, out_fp32=True)   # one 32-row matrix-core launch (17..32 rows)


@pytest.mark.parametrize("B", [2, 8])
def test_mfma_rows_kernel_7b_layers_full_size(B):
    """The 7B attention and MLP layers at full size with the default plan at B = 2 and 8 (the row-complete matrix-core
    kernel where it fits): sampled rows against the oracle."""
    from paper_2608_15602_amd import fluxbin as fb
    for spec in config_layers("c2_attn7b", "128") + config_layers("c3_mlp7b", "128"):
        L = make_layer(spec)
        packed = pack_layer(L)
        log(f"plan {spec.name} B={B}: {fb.fluxbin_plan_query(packed, B)['kernel_name']}")
        _parity(spec, B, rows=sample_rows(spec.M, 256, seed=B), packed=packed, L=L)
        del packed


PREFILL_SPECS = [
    LayerSpec("prefill_mu8", M=1536, N=2048, Kb=2, Ks=1, mu=8, S=61, g_r=128, g_s=61, seed=23),
    LayerSpec("prefill_mu4", M=700, N=1000, Kb=2, Ks=1, mu=4, S=40, g_r=128, g_s=40, seed=24),
    LayerSpec("prefill_fine", M=333, N=300, Kb=3, Ks=2, mu=8, S=77, g_r=64, g_s=8, seed=25),
]


@pytest.mark.parametrize("B", [17, 33, 40, 64, 65])
@pytest.mark.parametrize("spec", PREFILL_SPECS, ids=lambda s: s.name)
def test_prefill_batch_tiles(spec, B):
    """Batches above one launch's rows run as batch tiles (32 rows on layers with one row scale per chunk, else 16),
    one launch each: every row matches the oracle, and each tile's rows are bitwise those of a call on that tile's rows
    alone (a one-row tail runs a batch-1 kernel)."""
    from paper_2608_15602_amd import fluxbin as fb
    _, packed, x, y = _parity(spec, B, out_fp32=True)
    info = fb.fluxbin_plan_query(packed, B)
    tile = info["batch_tile_rows"]
    fine = (spec.g_r < 128 and spec.g_r < spec.N) or (spec.Ks > 0 and spec.S > 0 and spec.g_s < min(128, spec.S))
    assert tile == (16 if fine else 32), info
    assert info["batch_tiles"] == -(-B // tile), info
    for b0 in range(0, B, tile):
        part = run_gemm(packed, x[b0:b0 + tile], out_fp32=True)
        assert np.array_equal(part, y[b0:b0 + tile]), (B, b0)


TILE32_SPECS = [
    LayerSpec("tile32_mu8", M=2000, N=3000, Kb=2, Ks=1, mu=8, S=90, g_r=128, g_s=90, seed=31),
    LayerSpec("tile32_mu4", M=1100, N=2200, Kb=3, Ks=1, mu=4, S=33, g_r=128, g_s=33, seed=32),
    LayerSpec("tile32_1base", M=300, N=700, Kb=1, Ks=0, mu=8, S=0, g_r=128, g_s=1, seed=33),
]


@pytest.mark.parametrize("B", [17, 24, 32])
@pytest.mark.parametrize("spec", TILE32_SPECS, ids=lambda s: s.name)
def test_mfma_32_row_launch(spec, B):
    """17..32 batch rows in one matrix-core launch (two 16-row MFMA tiles per decoded sign operand): every row against
    the oracle, bitwise repeatable, and within tolerance of the same batch run as 16-row tiles."""
    from paper_2608_15602_amd import fluxbin as fb
    L = make_layer(spec)
    packed = pack_layer(L)
    info = fb.fluxbin_plan_query(packed, B)
    assert (info["kernel"], info["batch_tile_rows"], info["batch_tiles"]) == (3, 32, 1), info
    _, _, x, y = _parity(spec, B, packed=packed, L=L)
    assert np.array_equal(run_gemm(packed, x), y), "repeat differs"
    y16 = _with_env({"FLUXBIN_BATCH_TILE": "16"}, lambda: run_gemm(packed, x))
    _check(y, y16, "32-row launch vs 16-row tiles")


def test_mfma_32_row_launch_large_row_stride():
    """An x row stride so large that 15 strides pass 2^31 bytes (64-bit addressing of x): one 32-row launch gives
    bitwise the result of the same rows stored contiguously."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    spec = TILE32_SPECS[2]
    log("case 32-row launch, large x row stride")
    L = make_layer(spec)
    packed = pack_layer(L)
    B, ldx = 20, (1 << 30) // 15 + 64
    x = make_activations(L, B)
    flat = torch.zeros((B - 1) * ldx + spec.N, dtype=torch.float16, device="cuda")
    xs = flat.as_strided((B, spec.N), (ldx, 1))
    xs.copy_(x_tensor(x))
    y = fb.fluxbin_lut_gemm_smallbatch(packed, xs, out_fp32=True)
    torch.cuda.synchronize()
    y = y.cpu().numpy().astype(np.float64)
    del flat, xs
    assert np.array_equal(y, run_gemm(packed, x, out_fp32=True))
    _check(y, oracle.gemv_dense(L, x), "large row stride")


def test_prefill_batch_mlp70b_full_size():
    """A 64-row batch on the 70B MLP up layer at full size (two 32-row tiles on the matrix cores): sampled rows
    against the oracle."""
    spec = config_layers("c4_mlp70b", "128")[0]
    _parity(spec, 64, rows=sample_rows(spec.M, 96, seed=64))


@pytest.mark.parametrize("B", [4, 16])
def test_mfma_small_batch_mlp70b_full_size(B):
    """The matrix-core kernel on both 70B MLP layers at full size, in the launch configuration the benchmark times:
    sampled rows against the oracle, bitwise repeatable, and close to the LUT batch kernel's result."""
    import torch
    for spec in config_layers("c4_mlp70b", "128"):
        L = make_layer(spec)
        packed = pack_layer(L)
        rows = sample_rows(spec.M, 256, seed=B)
        _, _, x, y = _with_env(SMALL_BATCH_KERNELS["mfma"], lambda: _parity(spec, B, rows=rows, packed=packed, L=L))
        assert np.array_equal(_with_env(SMALL_BATCH_KERNELS["mfma"], lambda: run_gemm(packed, x)), y), "repeat differs"
        y_lut = _with_env(SMALL_BATCH_KERNELS["lut_batch"], lambda: run_gemm(packed, x))
        _check(y, y_lut, "matrix-core vs LUT batch kernel")
        del packed
        torch.cuda.empty_cache()


def test_strided_batch():
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    spec = LayerSpec("strided", M=700, N=512, Kb=2, Ks=1, mu=8, S=16, g_r=128, g_s=16, seed=23)
    log("case strided batch")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, 4)
    xt = torch.zeros(4, 600, dtype=torch.float16, device="cuda")
    xt[:, :512] = x_tensor(x)
    y = torch.full((4, 800), float("nan"), dtype=torch.float32, device="cuda")
    fb.fluxbin_lut_gemm_smallbatch(packed, xt[:, :512], y=y[:, :700], out_fp32=True)
    torch.cuda.synchronize()
    yc = y.cpu().numpy().astype(np.float64)
    assert np.all(np.isnan(yc[:, 700:]))
    _check(yc[:, :700], oracle.gemv_dense(L, x), "strided")


def test_strided_prefill_batch():
    """A 21-row batch (a 16-row tile and a 5-row tile) with row strides above N and M, fp16 and fp32 outputs: every
    row against the oracle and nothing written between the rows."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    spec = LayerSpec("strided_prefill", M=700, N=512, Kb=2, Ks=1, mu=8, S=16, g_r=128, g_s=16, seed=24)
    log("case strided prefill batch")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, 21)
    xt = torch.zeros(21, 601, dtype=torch.float16, device="cuda")
    xt[:, :512] = x_tensor(x)
    for fp32 in (True, False):
        y = torch.full((21, 777), float("nan"), dtype=torch.float32 if fp32 else torch.float16, device="cuda")
        fb.fluxbin_lut_gemm_smallbatch(packed, xt[:, :512], y=y[:, :700], out_fp32=fp32)
        torch.cuda.synchronize()
        yc = y.float().cpu().numpy().astype(np.float64)
        assert np.all(np.isnan(yc[:, 700:]))
        _check(yc[:, :700], oracle.gemv_dense(L, x), f"strided prefill fp32={fp32}")


def test_deterministic_and_exact_power_of_two_scaling():
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    spec = config_layers("c2_attn7b", "128")[0]
    log("case determinism + y(2x) == 2 y(x)")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, 1)
    ws = fb.make_workspace(packed, 1)
    y1 = run_gemm(packed, x, out_fp32=True, ws=ws)
    y2 = run_gemm(packed, x, out_fp32=True, ws=ws)
    assert np.array_equal(y1, y2)
    x2 = (oracle.f16_to_f64(x) * 2).astype(np.float16).view(np.uint16)
    y3 = run_gemm(packed, x2, out_fp32=True, ws=ws)
    assert np.array_equal(y3, 2 * y1)


def test_zero_activation_gives_zero():
    spec = LayerSpec("zero", M=512, N=512, Kb=2, Ks=1, mu=8, S=10, g_r=128, g_s=10, seed=24)
    log("case zero activations")
    L = make_layer(spec)
    packed = pack_layer(L)
    y = run_gemm(packed, np.zeros((1, 512), np.uint16), out_fp32=True)
    assert np.all(y == 0)


def test_stream_probe_runs_and_leaves_results_alone():
    """The measurement-only probe launches on every batch-1 plan shape (small and large layers) and writes nothing
    the GEMV reads: a GEMV after it gives the same result as before."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    log("case stream probe")
    sink = torch.zeros(256, dtype=torch.int32, device="cuda")
    for spec in (LayerSpec("p1", M=700, N=512, Kb=2, Ks=1, mu=8, S=9, g_r=128, g_s=9, seed=41),
                 LayerSpec("p2", M=4096, N=4096, Kb=2, Ks=1, mu=8, S=41, g_r=128, g_s=41, seed=42),
                 LayerSpec("p3", M=3000, N=1024, Kb=2, Ks=1, mu=4, S=20, g_r=128, g_s=20, seed=43)):
        L = make_layer(spec)
        packed = pack_layer(L)
        xb = make_activations(L, 1)
        y0 = run_gemm(packed, xb, out_fp32=True)
        fb.fluxbin_stream_probe(packed, sink)
        torch.cuda.synchronize()
        assert np.array_equal(run_gemm(packed, xb, out_fp32=True), y0)
    with pytest.raises(fb.FluxbinError):   # sink below 1024 bytes
        fb.fluxbin_stream_probe(packed, sink[:100])
    with fb.tuning(generic=1), pytest.raises(fb.FluxbinError):   # no split-tile batch-1 plan to follow
        fb.fluxbin_stream_probe(packed, sink)


def test_graph_replays_match_eager():
    """The kernels captured in a HIP graph give the eager result on every replay, with eager work in between."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    log("case graph replay")
    outs = []
    specs = [LayerSpec("g1", M=3000, N=2048, Kb=2, Ks=1, mu=8, S=70, g_r=128, g_s=70, seed=31),
             LayerSpec("g2", M=700, N=512, Kb=2, Ks=1, mu=4, S=9, g_r=512, g_s=9, seed=32),
             LayerSpec("g3", M=2000, N=1024, Kb=2, Ks=2, mu=8, S=128, g_r=64, g_s=16, seed=33, sal_block=128)]
    for spec in specs:
        L = make_layer(spec)
        packed = pack_layer(L)
        for B in (1, 3):
            x = x_tensor(make_activations(L, B))
            ws = fb.make_workspace(packed, B)
            y_eager = (fb.fluxbin_lut_gemv(packed, x[0], out_fp32=True, workspace=ws)[None] if B == 1 else
                       fb.fluxbin_lut_gemm_smallbatch(packed, x, out_fp32=True, workspace=ws)).clone()
            y = torch.empty_like(y_eager)
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                with torch.cuda.graph(g, stream=side):
                    if B == 1:
                        fb.fluxbin_lut_gemv(packed, x[0], y=y[0], out_fp32=True, workspace=ws)
                    else:
                        fb.fluxbin_lut_gemm_smallbatch(packed, x, y=y, out_fp32=True, workspace=ws)
            torch.cuda.current_stream().wait_stream(side)
            for r in range(4):
                y.fill_(float("nan"))
                g.replay()
                torch.cuda.synchronize()
                assert torch.equal(y, y_eager), (spec.name, B, r)
                fb.fluxbin_lut_gemv(packed, x[0], out_fp32=True, workspace=ws)   # eager work between replays
                torch.cuda.synchronize()


def test_workspace_shared_by_batch_sizes():
    """One workspace (the largest size queried) serves calls of one layer at every batch size and on every kernel, in
    any order: the tile counters of every launch plan lie in one region that no plan's partial sums cover, so each
    result equals the result on a fresh workspace."""
    import torch
    from paper_2608_15602_amd import fluxbin as fb
    log("case workspace shared by batch sizes")
    spec = LayerSpec("wsshare", M=3000, N=2048, Kb=2, Ks=1, mu=8, S=70, g_r=128, g_s=70, seed=33)
    L = make_layer(spec)
    packed = pack_layer(L)
    runs = [(1, {}), (3, {}), (2, {"FLUXBIN_MFMA": "0"}), (16, {}), (5, {"FLUXBIN_GENERIC": "1"}),
            (4, {"FLUXBIN_MFMA": "0"}), (1, {"FLUXBIN_NT": "1024", "FLUXBIN_ROWS": "0"}), (8, {"FLUXBIN_MFMA": "0"}),
            (1, {"FLUXBIN_ROWS": "1"}), (37, {})]
    n = max(_with_env(env, lambda: fb.fluxbin_workspace_query(packed, B)) for B, env in runs)
    shared = torch.empty((n + 255) // 256 * 256, dtype=torch.uint8, device="cuda")
    fb.fluxbin_workspace_init(shared)
    xs = {B: make_activations(L, B) for B, _ in runs}
    fresh = {i: _with_env(env, lambda: run_gemm(packed, xs[B], out_fp32=True, ws=fb.make_workspace(packed, B)))
             for i, (B, env) in enumerate(runs)}
    _check(fresh[1], oracle.gemv_dense(L, xs[3]), "B = 3 on a fresh workspace")
    for order in (runs, runs[::-1]):
        for B, env in order:
            i = runs.index((B, env))
            y = _with_env(env, lambda: run_gemm(packed, xs[B], out_fp32=True, ws=shared))
            assert np.array_equal(y, fresh[i]), (B, env)


@pytest.mark.parametrize("mu", [8, 4])
@pytest.mark.parametrize("B", [3, 8, 16])
def test_mfma_second_kernel_reduction_equals_counters(B, mu):
    """The matrix-core kernel's split tiles reduced by a second kernel (one workgroup per split tile and batch row) give
    the counter protocol's y bit for bit (same contributors, same order), on a layer with many contributors per tile,
    and match the oracle; so do workgroup ranges aligned to the row tiles (the default with the second kernel)."""
    from paper_2608_15602_amd import fluxbin as fb
    spec = LayerSpec("r2", M=3000, N=8192, Kb=3, Ks=1, mu=mu, S=100, g_r=128, g_s=100, seed=34)
    log(f"case second-kernel reduction B={B} mu={mu}")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, B)
    env = {"FLUXBIN_MFMA": "1", "FLUXBIN_MFMA_ROWS": "0", "FLUXBIN_ALIGN": "0"}
    y_c = _with_env({**env, "FLUXBIN_MFMA_R2": "0"},
                    lambda: run_gemm(packed, x, out_fp32=True, ws=fb.make_workspace(packed, B)))
    y_r = _with_env({**env, "FLUXBIN_MFMA_R2": "1"},
                    lambda: run_gemm(packed, x, out_fp32=True, ws=fb.make_workspace(packed, B)))
    assert np.array_equal(y_r, y_c), int(np.sum(y_r != y_c))
    y_ref = oracle.gemv_dense(L, x)
    _check(y_r, y_ref, "second-kernel reduction vs oracle")
    info = _with_env({**env, "FLUXBIN_ALIGN": "-1"}, lambda: fb.fluxbin_plan_query(packed, B))
    assert info["workgroups_per_tile"] > 1, info
    y_a = {}
    for r2 in ("0", "1"):
        y_a[r2] = _with_env({**env, "FLUXBIN_ALIGN": "-1", "FLUXBIN_MFMA_R2": r2},
                            lambda: run_gemm(packed, x, out_fp32=True, ws=fb.make_workspace(packed, B)))
    assert np.array_equal(y_a["1"], y_a["0"]), int(np.sum(y_a["1"] != y_a["0"]))
    _check(y_a["1"], y_ref, "tile-aligned ranges vs oracle")


# Unit ranges of the split-tile kernels: balanced over all units (FLUXBIN_ALIGN=0), aligned to row tiles where that
# fits one wave (-1, the default), and forced counts of workgroups per tile (k > 0: 1 = no split tiles; 3; a count
# that leaves some parts one unit longer than others).
ALIGN_CASES = [("batch1", 1, {"FLUXBIN_ROWS": "0"}), ("lut_batch", 3, {"FLUXBIN_MFMA": "0"}),
               ("lut_batch_r2", 2, {"FLUXBIN_MFMA": "0", "FLUXBIN_BAT_R2": "1"}),
               ("mfma", 5, {"FLUXBIN_MFMA": "1", "FLUXBIN_MFMA_ROWS": "0"}),
               ("mfma_counters", 9, {"FLUXBIN_MFMA": "1", "FLUXBIN_MFMA_ROWS": "0", "FLUXBIN_MFMA_R2": "0"})]


@pytest.mark.parametrize("case", ALIGN_CASES, ids=[c[0] for c in ALIGN_CASES])
@pytest.mark.parametrize("align", ["0", "-1", "1", "3", "7"])
def test_split_tile_unit_ranges(case, align):
    """Every split-tile kernel matches the oracle with balanced, tile-aligned and forced per-tile unit ranges (ragged
    last tile, a tile's parts of unequal length), and the plan reports the aligned split."""
    from paper_2608_15602_amd import fluxbin as fb
    name, B, env = case
    spec = LayerSpec("align", M=2600, N=1536, Kb=2, Ks=1, mu=8, S=150, g_r=128, g_s=150, seed=36)
    log(f"case unit ranges {name} B={B} align={align}")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, B)
    env = {**env, "FLUXBIN_ALIGN": align}
    info = _with_env(env, lambda: fb.fluxbin_plan_query(packed, B))
    if int(align) > 0:
        assert info["workgroups_per_tile"] == min(int(align), info["units"] // info["tiles"]) or \
            info["workgroups_per_tile"] > int(align), info   # raised to the kernel's unit cap
        assert info["workgroups"] == info["tiles"] * info["workgroups_per_tile"], info
    elif align == "0":
        assert info["workgroups_per_tile"] == 0, info
    y = _with_env(env, lambda: run_gemm(packed, x, out_fp32=True, ws=fb.make_workspace(packed, B)))
    _check(y, oracle.gemv_dense(L, x), f"{name} align {align}")
    y2 = _with_env(env, lambda: run_gemm(packed, x, out_fp32=True, ws=fb.make_workspace(packed, B)))
    assert np.array_equal(y2, y), "repeat differs"



@pytest.mark.parametrize("B", [2, 3, 4])
def test_lut_batch_second_kernel_reduction_equals_counters(B):
    """The LUT batch kernel's split tiles reduced by the second kernel give the counter protocol's y bit for bit, on a
    layer whose 1024-row tiles have about a hundred contributors each, and match the oracle."""
    from paper_2608_15602_amd import fluxbin as fb
    spec = LayerSpec("batr2", M=3000, N=8192, Kb=3, Ks=1, mu=8, S=100, g_r=128, g_s=100, seed=35)
    log(f"case LUT batch second-kernel reduction B={B}")
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, B)
    y = {}
    for align in ("0", "-1"):
        for r2 in ("0", "1"):
            y[r2] = _with_env({"FLUXBIN_MFMA": "0", "FLUXBIN_BAT_R2": r2, "FLUXBIN_ALIGN": align},
                              lambda: run_gemm(packed, x, out_fp32=True, ws=fb.make_workspace(packed, B)))
        assert np.array_equal(y["1"], y["0"]), (align, int(np.sum(y["1"] != y["0"])))
    _check(y["1"], oracle.gemv_dense(L, x), "LUT batch second-kernel reduction vs oracle")



# ------------------------------------------------------------------------------------------- fp16 subnormal inputs

def _subnormals(rng, shape):
    """Random fp16 subnormal bit patterns (nonzero exponent-0 values, random sign)."""
    mag = rng.integers(1, 1024, size=shape).astype(np.uint16)
    return (mag | (rng.integers(0, 2, size=shape).astype(np.uint16) << 15)).astype(np.uint16)


def _subnormal_case(which, mu):
    spec = LayerSpec(f"sub_{which}_mu{mu}", M=1500, N=1024, Kb=2, Ks=1, mu=mu, S=61, g_r=128, g_s=61, seed=70)
    L = make_layer(spec)
    rng = np.random.default_rng(71)
    B = 9
    x = make_activations(L, B)
    if which == "colscale":      # every global and salient column scale subnormal (positive: scales here are > 0)
        L.alpha_c[:] = _subnormals(rng, L.alpha_c.shape) & 0x7FFF
        L.alpha_sc[:] = _subnormals(rng, L.alpha_sc.shape) & 0x7FFF
    elif which == "rowscale":    # every row scale subnormal
        L.alpha_r[:] = _subnormals(rng, L.alpha_r.shape) & 0x7FFF
        L.alpha_sr[:] = _subnormals(rng, L.alpha_sr.shape) & 0x7FFF
    else:                        # every activation subnormal
        x = _subnormals(rng, x.shape)
    return L, x


@pytest.mark.parametrize("kernel", ["batch1", "rows", "lut_batch", "mfma", "mfma_rows"])
@pytest.mark.parametrize("which", ["colscale", "rowscale", "x"])
def test_fp16_subnormals_are_honoured(which, kernel):
    """Subnormal fp16 column scales, row scales or activations (the reading that subnormals are honoured on both
    sides): every product and sum stays far above the fp32 subnormal range, so a kernel that flushed fp16 subnormals
    to zero would return zeros. Batch 1, the LUT batch kernel at B = 3 and the matrix-core kernel at B = 3 and 9,
    against the fp64 oracle (fp32 output)."""
    L, x = _subnormal_case(which, 8)
    packed = pack_layer(L)
    env = {"batch1": {"FLUXBIN_ROWS": "0"}, "rows": {"FLUXBIN_ROWS": "1"}, "lut_batch": {"FLUXBIN_MFMA": "0"},
           "mfma": {"FLUXBIN_MFMA": "1", "FLUXBIN_MFMA_ROWS": "0"}, "mfma_rows": {"FLUXBIN_MFMA_ROWS": "1"}}[kernel]
    for B in ((1,) if kernel in ("batch1", "rows") else (3, 9) if kernel == "mfma" else (3, 8) if kernel == "mfma_rows"
              else (3,)):
        log(f"case subnormal {which} kernel={kernel} B={B}")
        xb = x[:B]
        y = _with_env(env, lambda: run_gemm(packed, xb, out_fp32=True))
        y_ref = oracle.gemv_dense(L, xb)
        assert np.abs(y_ref).max() > 0
        _check(y, y_ref, f"subnormal {which}, {kernel}, B={B}")


@pytest.mark.parametrize("which", ["colscale", "x"])
def test_fp16_subnormals_mu4(which):
    """The same at mu = 4 (batch-1 kernel, and the matrix cores at B = 3)."""
    L, x = _subnormal_case(which, 4)
    packed = pack_layer(L)
    for B in (1, 3):
        log(f"case subnormal mu4 {which} B={B}")
        y = run_gemm(packed, x[:B], out_fp32=True)
        _check(y, oracle.gemv_dense(L, x[:B]), f"subnormal mu4 {which} B={B}")


@pytest.mark.parametrize("kernel,B", [("lut_batch", 2), ("lut_batch", 4), ("mfma", 3), ("mfma", 16),
                                      ("mfma_rows", 3), ("mfma_rows", 8), ("generic", 3)])
def test_small_batch_power_of_two_scaling_is_exact(kernel, B):
    """y(2x) == 2 y(x) bit for bit on the small-batch kernels (scaling by two commutes with every fp32 rounding when
    nothing overflows or underflows), and repeated calls are bitwise equal."""
    spec = LayerSpec("pow2", M=3000, N=2048, Kb=2, Ks=1, mu=8, S=70, g_r=128, g_s=70, seed=72)
    L = make_layer(spec)
    packed = pack_layer(L)
    x = make_activations(L, B)
    x2 = (oracle.f16_to_f64(x) * 2).astype(np.float16).view(np.uint16)
    env = {"lut_batch": {"FLUXBIN_MFMA": "0"}, "mfma": {"FLUXBIN_MFMA": "1", "FLUXBIN_MFMA_ROWS": "0"},
           "mfma_rows": {"FLUXBIN_MFMA_ROWS": "1"}, "generic": {"FLUXBIN_GENERIC": "1"}}[kernel]
    log(f"case y(2x) == 2 y(x) {kernel} B={B}")
    y1 = _with_env(env, lambda: run_gemm(packed, x, out_fp32=True))
    y1b = _with_env(env, lambda: run_gemm(packed, x, out_fp32=True))
    y2 = _with_env(env, lambda: run_gemm(packed, x2, out_fp32=True))
    assert np.array_equal(y1, y1b)
    assert np.array_equal(y2, 2 * y1), int(np.sum(y2 != 2 * y1))
