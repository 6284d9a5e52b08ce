"""Synthetic Llama-shaped FluxBin layers.

The paper measures on LLaMA-2/3.1 and Qwen3 layers (Sec. 4, App. E.4). No weights or datasets are available, so
these seeded layers stand in for them, with the same shapes and with the format of Sec. 3.1:
  * ``signs``      uint32 [Kb, M, W]  canonical packed sign planes B^(k), W = ceil(N/32); bit t of word w is column
                   32w+t, a set bit means +1. Bits past column N-1 are zero.
  * ``alpha_r``    uint16 [Kb, M, G_r] fp16 row scales, one per (row, group of g_r columns), G_r = ceil(N/g_r).
  * ``alpha_c``    uint16 [Kb, N]      fp16 column scales.
  * ``sal_idx``    int32  [S]          salient column indices, strictly increasing.
  * ``sal_signs``  uint32 [Ks, M, W]   full-width salient sign planes B_s^(k) (bits off the salient set are random
                   and must be ignored).
  * ``alpha_sr``   uint16 [Ks, M, G_s] fp16 salient row scales, one per (row, group of g_s salient columns).
  * ``alpha_sc``   uint16 [Ks, N]      fp16 full-width salient column scales.
  * ``x``          uint16 [B, N]       fp16 activations.

Distributions: signs Bernoulli(1/2); row scales fp16(|N(0, 0.05)|); column scales fp16(lognormal(0, 0.3));
activations fp16(N(0, 1)) with an optional fraction of outlier channels multiplied by 20 before rounding; salient
columns drawn uniformly without replacement. fp16 values are produced by round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List

import numpy as np


def _round_half_up(v: float) -> int:
    return int(math.floor(v + 0.5))


def salient_count(N: int, frac: float) -> int:
    """Number of salient columns for a fraction of N (fractional counts round half up)."""
    return _round_half_up(frac * N)


@dataclasses.dataclass(frozen=True)
class LayerSpec:
    name: str
    M: int            # output channels (rows of W)
    N: int            # input channels (columns of W)
    Kb: int           # global binary bases
    Ks: int           # salient binary bases
    mu: int           # LUT sub-vector length (4 or 8)
    S: int            # number of salient columns
    g_r: int          # row-scale group (columns) of the global branch
    g_s: int          # row-scale group (salient columns) of the salient branch
    outlier_frac: float = 0.0
    seed: int = 0
    layer_id: int = 0
    sal_block: int = 0   # > 0: the paper's structured selection, S / ceil(N / sal_block) columns in every block of
                         # sal_block input columns (else S columns drawn uniformly over all N)

    @property
    def G_r(self) -> int:
        return -(-self.N // self.g_r)

    @property
    def G_s(self) -> int:
        return -(-self.S // self.g_s) if self.S > 0 else 0

    @property
    def W(self) -> int:
        return -(-self.N // 32)

    def with_(self, **kw) -> "LayerSpec":
        return dataclasses.replace(self, **kw)


@dataclasses.dataclass
class SyntheticLayer:
    spec: LayerSpec
    signs: np.ndarray
    alpha_r: np.ndarray
    alpha_c: np.ndarray
    sal_idx: np.ndarray
    sal_signs: np.ndarray
    alpha_sr: np.ndarray
    alpha_sc: np.ndarray
    outliers: np.ndarray


def _f16_bits(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a.astype(np.float16)).view(np.uint16)


def _random_sign_words(rng: np.random.Generator, planes: int, M: int, N: int) -> np.ndarray:
    nbytes = -(-N // 8)
    W = -(-N // 32)
    raw = np.frombuffer(rng.bytes(planes * M * nbytes), dtype=np.uint8).reshape(planes, M, nbytes)
    buf = np.zeros((planes, M, W * 4), dtype=np.uint8)
    buf[:, :, :nbytes] = raw
    if N % 8:
        buf[:, :, nbytes - 1] &= np.uint8((1 << (N % 8)) - 1)
    return buf.view("<u4").reshape(planes, M, W).astype(np.uint32, copy=False)


def make_layer(spec: LayerSpec) -> SyntheticLayer:
    """Draw one layer. The draw order is fixed: global signs, alpha_r, alpha_c, salient set, salient signs,
    alpha_sr, alpha_sc, outlier channels."""
    rng = np.random.default_rng([spec.seed, spec.layer_id])
    M, N, Kb, Ks, S = spec.M, spec.N, spec.Kb, spec.Ks, spec.S
    signs = _random_sign_words(rng, Kb, M, N)
    alpha_r = _f16_bits(np.abs(rng.normal(0.0, 0.05, size=(Kb, M, spec.G_r))))
    alpha_c = _f16_bits(rng.lognormal(0.0, 0.3, size=(Kb, N)))
    if S > 0 and spec.sal_block > 0:
        nb = -(-N // spec.sal_block)
        per = S // nb
        if per * nb != S:
            raise ValueError("structured selection needs S = s * ceil(N / sal_block)")
        parts = []
        for b0 in range(0, N, spec.sal_block):
            cols = np.arange(b0, min(N, b0 + spec.sal_block))
            parts.append(np.sort(rng.choice(cols, size=min(per, cols.size), replace=False)))
        sal_idx = np.concatenate(parts).astype(np.int32)
    elif S > 0:
        sal_idx = np.sort(rng.choice(N, size=S, replace=False)).astype(np.int32)
    else:
        sal_idx = np.zeros(0, np.int32)
    sal_signs = _random_sign_words(rng, Ks, M, N)
    alpha_sr = _f16_bits(np.abs(rng.normal(0.0, 0.05, size=(Ks, M, spec.G_s))))
    alpha_sc = _f16_bits(rng.lognormal(0.0, 0.3, size=(Ks, N)))
    n_out = _round_half_up(spec.outlier_frac * N)
    outliers = np.sort(rng.choice(N, size=n_out, replace=False)).astype(np.int64) if n_out else np.zeros(0, np.int64)
    return SyntheticLayer(spec, signs, alpha_r, alpha_c, sal_idx, sal_signs, alpha_sr, alpha_sc, outliers)


def vcm_off_equivalent(layer: SyntheticLayer) -> SyntheticLayer:
    """The same weights without the dense salient repack (the paper's VCM ablation): the Ks salient bases become Ks
    more global bases over all N columns, with their full-width sign planes as stored, a column scale that is zero off
    the salient set, and the one salient row scale of each row repeated over the row-scale groups. Only valid when a
    row has one salient row scale per base (g_s >= S, as in every workload here). Same activations (same seed, layer
    id and outlier channels); same exact result."""
    sp = layer.spec
    if sp.S > 0 and sp.g_s < sp.S:
        raise ValueError("vcm_off_equivalent needs one salient row scale per row and base (g_s >= S)")
    ks = sp.Ks if sp.S > 0 else 0
    spec = sp.with_(name=sp.name + "_vcmoff", Kb=sp.Kb + ks, Ks=0, S=0, g_s=1)
    G = spec.G_r
    signs = np.concatenate([layer.signs, layer.sal_signs[:ks]], axis=0)
    ar_sal = (np.repeat(layer.alpha_sr[:ks, :, :1], G, axis=2) if ks
              else np.zeros((0, sp.M, G), dtype=layer.alpha_r.dtype))
    alpha_r = np.concatenate([layer.alpha_r, ar_sal], axis=0)
    ac_sal = np.zeros((ks, sp.N), dtype=np.uint16)
    if ks:
        ac_sal[:, layer.sal_idx] = layer.alpha_sc[:ks, layer.sal_idx]
    alpha_c = np.concatenate([layer.alpha_c, ac_sal], axis=0)
    W = -(-sp.N // 32)
    return SyntheticLayer(spec, np.ascontiguousarray(signs), np.ascontiguousarray(alpha_r),
                          np.ascontiguousarray(alpha_c), np.zeros(0, np.int32), np.zeros((0, sp.M, W), np.uint32),
                          np.zeros((0, sp.M, 1), np.uint16), np.zeros((0, sp.N), np.uint16), layer.outliers)


def make_activations(layer: SyntheticLayer, B: int, draw: int = 0) -> np.ndarray:
    """fp16 activations [B, N] (as uint16 bits); outlier channels scaled by 20 before rounding."""
    spec = layer.spec
    rng = np.random.default_rng([spec.seed, spec.layer_id, 1000 + B, draw])
    x = rng.normal(0.0, 1.0, size=(B, spec.N))
    if layer.outliers.size:
        x[:, layer.outliers] *= 20.0
    return _f16_bits(x)


def paper_config(name: str, M: int, N: int, Kb: int, s: int = 0, g: int = 128, mu: int = 8, seed: int = 7,
                 layer_id: int = 0) -> LayerSpec:
    """A layer in the paper's {Kb-sS-gG} configuration (Sec. 4, App. C.2): Kb global bases with one row scale per
    (row, block of g columns); with s > 0 also Ks = Kb salient bases on s columns of every block of g (structured
    selection, Sec. 3.1), each salient base with one row scale per (row, block), i.e. per s VCM dense columns."""
    if s == 0:
        return LayerSpec(name, M=M, N=N, Kb=Kb, Ks=0, mu=mu, S=0, g_r=g, g_s=1, seed=seed, layer_id=layer_id)
    S = s * (-(-N // g))
    return LayerSpec(name, M=M, N=N, Kb=Kb, Ks=Kb, mu=mu, S=S, g_r=g, g_s=s, seed=seed, layer_id=layer_id,
                     sal_block=g)


def kernel_latency_layers() -> List[LayerSpec]:
    """The operator shapes and configurations of the paper's kernel-latency table (App. E.4): out x in 4096x4096,
    5120x5120, 4096x11008 and 5120x13824, each as 2b-g128, 2b-s8-g128, 2b-s16-g128 and 4b-g128."""
    out = []
    lid = 200
    for M, N in ((4096, 4096), (5120, 5120), (4096, 11008), (5120, 13824)):
        for tag, Kb, s in (("2b", 2, 0), ("2b-s8", 2, 8), ("2b-s16", 2, 16), ("4b", 4, 0)):
            out.append(paper_config(f"{M}x{N}_{tag}-g128", M, N, Kb, s, 128, layer_id=lid))
            lid += 1
    return out


def _attn_mlp(name, M, N, Kb, frac, seed, layer_id, mu=8, g_r=128, outlier_frac=0.0):
    S = salient_count(N, frac)
    return LayerSpec(name=name, M=M, N=N, Kb=Kb, Ks=1, mu=mu, S=S, g_r=g_r, g_s=max(S, 1),
                     outlier_frac=outlier_frac, seed=seed, layer_id=layer_id)


def config_layers(cfg: str, g_r: str = "128") -> List[LayerSpec]:
    """Layers of one workload. ``g_r`` is "128" (one row scale per 128 columns) or "N" (one per row)."""
    specs = CONFIGS[cfg]["layers"]
    out = []
    for s in specs:
        gr = s.g_r if g_r == "128" else s.N
        out.append(s.with_(g_r=gr))
    return out


def kernel_variant_layers(g_r: str = "128") -> List[LayerSpec]:
    """The 70B MLP up shape (28672 x 8192, out x in) in the kernel variants the paper ablates: mu = 8 and mu = 4 with
    3 bases + 1 salient base on 5% of the columns, pure global bases (3 and 4, no salient part), and 2 bases + 1 on 1%
    of the columns. Used for timing and for sampled-row parity at full size."""
    M, N = 28672, 8192
    out = [_attn_mlp("hyb3b5_mu8", M, N, 3, 0.05, seed=3, layer_id=10, outlier_frac=0.001),
           _attn_mlp("hyb3b5_mu4", M, N, 3, 0.05, seed=3, layer_id=11, mu=4, outlier_frac=0.001),
           LayerSpec("glob3b_mu8", M=M, N=N, Kb=3, Ks=0, mu=8, S=0, g_r=128, g_s=1, outlier_frac=0.001, seed=3,
                     layer_id=12),
           LayerSpec("glob4b_mu8", M=M, N=N, Kb=4, Ks=0, mu=8, S=0, g_r=128, g_s=1, outlier_frac=0.001, seed=3,
                     layer_id=13),
           _attn_mlp("hyb2b1_mu8", M, N, 2, 0.01, seed=3, layer_id=14, outlier_frac=0.001)]
    return [s.with_(g_r=s.N) if g_r == "N" else s for s in out]


def shard_layers(P: int, g_r: str = "128") -> List[LayerSpec]:
    """One rank's share of the 70B MLP layers when P ranks split them: the up projection by output rows
    (28672 / P x 8192, every input column, the same 5% salient columns) and the down projection by input columns
    (8192 x 28672 / P, the salient columns that fall in the rank's column range: 5% of them, drawn like any other
    layer's). These are the layers one GPU runs when the path is sharded; their partial outputs would then be
    concatenated (up) or summed across ranks (down)."""
    out = [_attn_mlp(f"up_p{P}", 28672 // P, 8192, 3, 0.05, seed=6, layer_id=200 + 2 * P, outlier_frac=0.001),
           _attn_mlp(f"down_p{P}", 8192, 28672 // P, 3, 0.05, seed=6, layer_id=201 + 2 * P, outlier_frac=0.001)]
    return [s.with_(g_r=s.N) if g_r == "N" else s for s in out]


def fused_decoder_layers(g_r: str = "128") -> List[LayerSpec]:
    """The 70B decoder layer's linears with the launches that share an input fused by stacking output rows: q, k and v
    as one 10240 x 8192 layer, gate and up as one 57344 x 8192 layer, then o and down. A fused layer has one salient
    column set (the stacked rows read the same input columns), drawn like any other layer. Both hybrid variants."""
    out = []
    lid = 100
    for variant, Kb, frac in (("2b1pct", 2, 0.01), ("3b5pct", 3, 0.05)):
        for nm, M, N in (("qkv", 10240, 8192), ("o", 8192, 8192), ("gate_up", 57344, 8192), ("down", 8192, 28672)):
            out.append(_attn_mlp(f"{variant}_{nm}", M, N, Kb, frac, seed=4, layer_id=lid, outlier_frac=0.001))
            lid += 1
    return [s.with_(g_r=s.N) if g_r == "N" else s for s in out]


def _build_configs() -> Dict[str, dict]:
    c = {}
    c["c1_tiny"] = dict(
        desc="tiny single linear 512x256 (out x in), 2 bases + 1 salient base on 8 columns, mu=4, batch 1",
        batches=[1],
        layers=[LayerSpec("tiny", M=512, N=256, Kb=2, Ks=1, mu=4, S=8, g_r=128, g_s=8, seed=0, layer_id=0)],
    )
    c["c2_attn7b"] = dict(
        desc="Llama-7B attention projection 4096x4096, 2 bases + 1 on 2% salient columns, mu=8, batch 1",
        batches=[1],
        layers=[_attn_mlp("attn_proj", 4096, 4096, 2, 0.02, seed=1, layer_id=0)],
    )
    c["c3_mlp7b"] = dict(
        desc="Llama-7B MLP gate/up 11008x4096 and down 4096x11008, 2 bases + 1 on 3% salient, mu=8, batch 1-8",
        batches=[1, 2, 4, 8],
        layers=[_attn_mlp("gate_up", 11008, 4096, 2, 0.03, seed=2, layer_id=0),
                _attn_mlp("down", 4096, 11008, 2, 0.03, seed=2, layer_id=1)],
    )
    c["c4_mlp70b"] = dict(
        desc="70B-shaped MLP up 28672x8192 and down 8192x28672, 3 bases + 1 on 5% salient, mu=8, batch 1, "
             "0.1% outlier channels x20",
        batches=[1],
        layers=[_attn_mlp("up", 28672, 8192, 3, 0.05, seed=3, layer_id=0, outlier_frac=0.001),
                _attn_mlp("down", 8192, 28672, 3, 0.05, seed=3, layer_id=1, outlier_frac=0.001)],
    )
    layers5 = []
    lid = 0
    for variant, Kb, frac in (("2b1pct", 2, 0.01), ("3b5pct", 3, 0.05)):
        for nm, M, N in (("q", 8192, 8192), ("k", 1024, 8192), ("v", 1024, 8192), ("o", 8192, 8192),
                         ("gate", 28672, 8192), ("up", 28672, 8192), ("down", 8192, 28672)):
            layers5.append(_attn_mlp(f"{variant}_{nm}", M, N, Kb, frac, seed=4, layer_id=lid, outlier_frac=0.001))
            lid += 1
    c["c5_layer70b"] = dict(
        desc="70B decoder-layer linears (q,k,v,o with GQA, gate, up, down), 2b/1% and 3b/5% hybrid, batch 1/4/16",
        batches=[1, 4, 16],
        layers=layers5,
    )
    return c


CONFIGS = _build_configs()


def make_weight_matrix(M: int, N: int, seed: int, outlier_frac: float = 0.01, outlier_scale: float = 10.0):
    """A dense fp32 weight matrix [M, N] for the decomposition: N(0, 0.02) entries, with round_half_up(frac * N)
    uniformly chosen outlier columns scaled by outlier_scale (the column-clustered outliers the saliency search is
    for), and a synthetic diagonal inverse Hessian [N] drawn uniform(0.5, 2.0). Draw order: entries, outlier columns,
    Hessian diagonal, from numpy.random.default_rng([seed, 9000])."""
    rng = np.random.default_rng([seed, 9000])
    W = rng.normal(0.0, 0.02, size=(M, N))
    n_out = salient_count(N, outlier_frac)
    cols = rng.choice(N, size=n_out, replace=False) if n_out > 0 else np.zeros(0, dtype=np.int64)
    W[:, cols] *= outlier_scale
    hinv = rng.uniform(0.5, 2.0, size=N)
    return W.astype(np.float32), hinv

