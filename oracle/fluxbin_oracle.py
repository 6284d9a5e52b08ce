"""FluxBin hot-path oracle: plain, slow, fp64 CPU reference of what the LUT-GEMV computes.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this package. It shares no code with the HIP path (``paper_2608_15602_amd/``) and never imports it.

Paper: FluxBin (arXiv 2608.15602). Equation numbers are the paper's:
  (3)  row-column binary decomposition  W^(k) = (alpha_r^(k) alpha_c^(k)^T) * B^(k), with one row scale per group
       of columns (Sec. 3.1);
  (9)  hybrid bases: global bases plus salient bases restricted to the salient-column mask (Sec. 3.1);
  (10) the hybrid GEMV  X W^T  split into a global and a salient term (Sec. 3.2);
  (11) column scales folded into the activation, row scales applied after the binary product (Sec. 3.2);
  (12) VCM dense extraction of the salient sign columns, (13) gather of X_sal and alpha_scd (Sec. 3.2, Def. VCM);
  (14) LUT-BSF: LUT[p] = sum_n (x_sub[n] alpha_c,sub[n]) (2 b_n(p) - 1) (Sec. 3.2, Def. LUT-BSF);
  (15) LUT reading with row scales, for the global and the VCM salient term (Sec. 3.2).

Readings where the paper is silent or ambiguous:
  * bit n of a pattern p (n = 0..mu-1) belongs to the n-th element of the sub-vector (LSB first); a set bit is +1;
  * row scales: one per (row, group of g_r consecutive columns); salient row scales: one per (row, group of g_s
    consecutive VCM dense columns);
  * a sub-vector that runs past the end of the columns is padded with zero activations, which contribute nothing.

Two independent routes are given: ``gemv_dense`` reconstructs W-hat explicitly (the definition) and multiplies;
``gemv_lut`` follows the kernel's algorithm (VCM, LUT-BSF, LUT reading, row scale). They agree in exact arithmetic.
"""
from __future__ import annotations

from typing import Dict, Iterable, Optional, Tuple

import numpy as np


# ----------------------------------------------------------------------------------------------------------------
# Input decoding
# ----------------------------------------------------------------------------------------------------------------

def f16_to_f64(bits) -> np.ndarray:
    """IEEE binary16 bit patterns (uint16) to float64. Exact, subnormals included."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def sign_bits(words: np.ndarray, N: int) -> np.ndarray:
    """Canonical packed planes [..., W] uint32 -> bits [..., N] in {0, 1}.

    Bit t of word w is column 32w + t (little-endian words, LSB first)."""
    w = np.ascontiguousarray(np.asarray(words, dtype=np.uint32).astype("<u4"))
    b = np.unpackbits(w.view(np.uint8), axis=-1, bitorder="little")
    return b[..., :N]


def sign_pm1(words: np.ndarray, N: int) -> np.ndarray:
    """Canonical packed planes -> {-1, +1} as float64, by the bit-to-sign map (2b - 1) of Eq. (14)."""
    return 2.0 * sign_bits(words, N).astype(np.float64) - 1.0


# ----------------------------------------------------------------------------------------------------------------
# Route 1: the definition. Reconstruct W-hat and multiply (Eqs. 3, 9, 10).
# ----------------------------------------------------------------------------------------------------------------

def reconstruct_rows(L, r0: int, r1: int) -> np.ndarray:
    """Rows [r0, r1) of W-hat in float64.

    Global term, Eq. (3) summed over k with one row scale per group (Sec. 3.1):
        W[i, j] = sum_k alpha_r^(k)[i, j // g_r] * alpha_c^(k)[j] * B^(k)[i, j]
    Salient refinement, Eq. (9): for the t-th salient column j = I_sal[t] add
        sum_k alpha_sr^(k)[i, t // g_s] * alpha_sc^(k)[j] * B_s^(k)[i, j]
    """
    s = L.spec
    N = s.N
    cols = np.arange(N)
    W = np.zeros((r1 - r0, N), dtype=np.float64)
    for k in range(s.Kb):
        B = sign_pm1(L.signs[k, r0:r1], N)
        ar = f16_to_f64(L.alpha_r[k, r0:r1])[:, cols // s.g_r]
        ac = f16_to_f64(L.alpha_c[k])[None, :]
        W += ar * ac * B
    if s.S > 0:
        idx = np.asarray(L.sal_idx, dtype=np.int64)
        t = np.arange(s.S)
        for k in range(s.Ks):
            Bs = sign_pm1(L.sal_signs[k, r0:r1], N)[:, idx]
            asr = f16_to_f64(L.alpha_sr[k, r0:r1])[:, t // s.g_s]
            asc = f16_to_f64(L.alpha_sc[k])[idx][None, :]
            W[:, idx] += asr * asc * Bs
    return W


def gemv_dense(L, x_bits: np.ndarray, rows: Optional[Iterable[int]] = None, block: int = 256,
               row_range: Optional[Tuple[int, int]] = None) -> np.ndarray:
    """y*[b, i] = sum_j W-hat[i, j] x[b, j] in float64 (Eq. 10), by explicit reconstruction in row blocks.

    ``rows`` restricts the output to a sorted subset of rows (the result then has one column per listed row);
    ``row_range`` = (r0, r1) to the contiguous rows r0 <= i < r1."""
    x = f16_to_f64(x_bits)
    if x.ndim == 1:
        x = x[None, :]
    M = L.spec.M
    if rows is None:
        lo, hi = row_range if row_range is not None else (0, M)
        out = np.zeros((x.shape[0], hi - lo), dtype=np.float64)
        for r0 in range(lo, hi, block):
            r1 = min(hi, r0 + block)
            out[:, r0 - lo:r1 - lo] = (reconstruct_rows(L, r0, r1) @ x.T).T
        return out
    rows = np.asarray(list(rows), dtype=np.int64)
    out = np.zeros((x.shape[0], rows.size), dtype=np.float64)
    for n, i in enumerate(rows):
        out[:, n] = reconstruct_rows(L, int(i), int(i) + 1)[0] @ x.T
    return out


# ----------------------------------------------------------------------------------------------------------------
# Route 2: the kernel's algorithm in float64 (Eqs. 11-15).
# ----------------------------------------------------------------------------------------------------------------

def pattern_signs(mu: int) -> np.ndarray:
    """Matrix [2^mu, mu] of (2 b_n(p) - 1): row p, column n is +1 if bit n of p is set, else -1 (Eq. 14)."""
    p = np.arange(1 << mu)[:, None]
    n = np.arange(mu)[None, :]
    return (2 * ((p >> n) & 1) - 1).astype(np.float64)


def lut_bsf(x_sub: np.ndarray, a_sub: np.ndarray) -> np.ndarray:
    """LUT with scale fusion, Eq. (14): LUT[p] = sum_n (x_sub[n] * alpha_sub[n]) * (2 b_n(p) - 1).

    ``x_sub``/``a_sub`` are [..., mu]; the result is [..., 2^mu]."""
    mu = x_sub.shape[-1]
    xc = x_sub * a_sub
    return xc @ pattern_signs(mu).T


def patterns(bits: np.ndarray, mu: int) -> np.ndarray:
    """mu-bit patterns p of consecutive column runs: bits [..., n_cols] -> p [..., ceil(n_cols/mu)].

    Element n of a sub-vector is bit n of p. A run shorter than mu at the end is padded with zero bits."""
    n_cols = bits.shape[-1]
    n_sub = -(-n_cols // mu)
    pad = n_sub * mu - n_cols
    if pad:
        bits = np.concatenate([bits, np.zeros(bits.shape[:-1] + (pad,), dtype=bits.dtype)], axis=-1)
    b = bits.reshape(bits.shape[:-1] + (n_sub, mu)).astype(np.int64)
    return (b << np.arange(mu)).sum(axis=-1)


def _subvectors(v: np.ndarray, mu: int) -> np.ndarray:
    """[..., n] -> [..., ceil(n/mu), mu] with zero padding at the end (padding contributes nothing)."""
    n = v.shape[-1]
    n_sub = -(-n // mu)
    pad = n_sub * mu - n
    if pad:
        v = np.concatenate([v, np.zeros(v.shape[:-1] + (pad,), dtype=v.dtype)], axis=-1)
    return v.reshape(v.shape[:-1] + (n_sub, mu))


def vcm_dense_bits(L) -> np.ndarray:
    """Eq. (12): dense salient planes B_sd^(k) = the salient columns of B_s^(k), in I_sal order. [Ks, M, S] bits."""
    idx = np.asarray(L.sal_idx, dtype=np.int64)
    return sign_bits(L.sal_signs, L.spec.N)[:, :, idx]


def vcm_gather(L, x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. (13): X_sal = X[:, I_sal] and alpha_scd^(k) = alpha_sc^(k)[I_sal] (float64)."""
    idx = np.asarray(L.sal_idx, dtype=np.int64)
    return x[:, idx], f16_to_f64(L.alpha_sc)[:, idx]


def _lut_branch(bits: np.ndarray, x: np.ndarray, a_col: np.ndarray, a_row: np.ndarray, g: int, mu: int) -> np.ndarray:
    """One base of one branch. bits [M, n], x [B, n], a_col [n], a_row [M, G] -> [B, M].

    Builds one LUT per sub-vector from x * alpha_col (Eq. 14), reads it at each row's pattern, sums the reads of each
    row-scale group and multiplies the sum by that group's row scale (Eq. 15)."""
    M, n = bits.shape
    p = patterns(bits, mu)                                   # [M, n_sub]
    n_sub = p.shape[1]
    xs = _subvectors(x, mu)                                  # [B, n_sub, mu]
    asub = _subvectors(a_col[None, :], mu)[0]                # [n_sub, mu]
    lut = lut_bsf(xs, asub[None])                            # [B, n_sub, 2^mu]
    reads = np.take_along_axis(lut[:, None, :, :], p[None, :, :, None], axis=-1)[..., 0]   # [B, M, n_sub]
    group = (np.arange(n_sub) * mu) // g                     # row-scale group of each sub-vector
    G = a_row.shape[1]
    y = np.zeros((x.shape[0], M), dtype=np.float64)
    for q in range(G):
        sel = group == q
        if sel.any():
            y += reads[:, :, sel].sum(axis=-1) * a_row[None, :, q]
    return y


def gemv_lut(L, x_bits: np.ndarray) -> np.ndarray:
    """y via the LUT algorithm in float64: Eq. (11) column-scale folding, Eqs. (12)-(13) VCM for the salient term,
    Eq. (14) LUT-BSF and Eq. (15) LUT reading with row scales. [B, M]."""
    s = L.spec
    x = f16_to_f64(x_bits)
    if x.ndim == 1:
        x = x[None, :]
    if s.g_r % s.mu and s.g_r < s.N:
        raise ValueError("a row-scale group must hold whole sub-vectors")
    if s.S > 0 and s.g_s % s.mu and s.g_s < s.S:
        raise ValueError("a salient row-scale group must hold whole sub-vectors")
    y = np.zeros((x.shape[0], s.M), dtype=np.float64)
    bits = sign_bits(L.signs, s.N)
    for k in range(s.Kb):
        y += _lut_branch(bits[k], x, f16_to_f64(L.alpha_c[k]), f16_to_f64(L.alpha_r[k]), s.g_r, s.mu)
    if s.S > 0 and s.Ks > 0:
        dense = vcm_dense_bits(L)
        x_sal, a_scd = vcm_gather(L, x)
        for k in range(s.Ks):
            y += _lut_branch(dense[k], x_sal, a_scd[k], f16_to_f64(L.alpha_sr[k]), s.g_s, s.mu)
    return y


def lut_indices(L) -> Dict[str, np.ndarray]:
    """The pattern p read for every (base, row, sub-vector): global [Kb, M, ceil(N/mu)] and salient (over the VCM dense
    columns) [Ks, M, ceil(S/mu)]."""
    s = L.spec
    out = {"global": patterns(sign_bits(L.signs, s.N), s.mu)}
    if s.S > 0 and s.Ks > 0:
        out["salient"] = patterns(vcm_dense_bits(L), s.mu)
    else:
        out["salient"] = np.zeros((s.Ks, s.M, 0), dtype=np.int64)
    return out


# ----------------------------------------------------------------------------------------------------------------
# Parity rule
# ----------------------------------------------------------------------------------------------------------------

def parity_check(y: np.ndarray, y_ref: np.ndarray, rel: float = 2e-3, floor: float = 1e-3) -> Dict[str, float]:
    """Per-element rule |y - y*| <= rel * max(|y*|, floor * max|y*| of that batch row).

    Plain per-element relative error is ill-posed for outputs that are sums of random signs (some are ~0), so the
    bound is floored at a fraction of the row's infinity norm. Returns statistics and ``ok``."""
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    if y_ref.ndim == 1:
        y, y_ref = y[None], y_ref[None]
    inf = np.abs(y_ref).max(axis=-1, keepdims=True) if y_ref.size else np.zeros((y_ref.shape[0], 1))
    bound = rel * np.maximum(np.abs(y_ref), floor * inf)
    err = np.abs(y - y_ref)
    ok = bool(np.all(np.isfinite(y)) and np.all(err <= bound))
    big = np.abs(y_ref) >= floor * inf
    with np.errstate(divide="ignore", invalid="ignore"):
        normwise = float((err.max(axis=-1, keepdims=True) / np.where(inf > 0, inf, 1)).max()) if y.size else 0.0
        rel_big = float((err[big] / np.abs(y_ref[big])).max()) if big.any() else 0.0
        worst = float((err / np.where(bound > 0, bound, 1)).max()) if y.size else 0.0
    return {"ok": ok, "normwise": normwise, "max_rel_above_floor": rel_big, "worst_bound_ratio": worst}


# ----------------------------------------------------------------------------------------------------------------
# Cost formulas printed in the paper (App. C.1, C.2, E.2, E.3)
# ----------------------------------------------------------------------------------------------------------------

def complexity(M: int, N: int, N_sal: int, Kb: int, Ks: int, mu: int) -> Dict[str, float]:
    """LUT build and read operation counts (App. C.1): C_build = 2^mu/mu (Kb N + Ks N_sal),
    C_read = M/mu (Kb N + Ks N_sal)."""
    work = Kb * N + Ks * N_sal
    return {"build": (2 ** mu) / mu * work, "read": M / mu * work}


def storage_bits(M: int, N: int, Kb: int, Ks: int, g: int, s: int) -> float:
    """Total storage in bits (App. C.2): S_base = Kb (M N + 16 N + 16 M N/g);
    S_sal = Ks (M N_sal + 16 N_sal + 16 M N/g) + 16 N_sal with N_sal = (N/g) s. Pure global when s = 0 (no salient
    branch at all)."""
    S_base = Kb * (M * N + 16 * N + 16 * M * N / g)
    if s == 0:
        return S_base
    N_sal = (N / g) * s
    S_sal = Ks * (M * N_sal + 16 * N_sal + 16 * M * N / g) + 16 * N_sal
    return S_base + S_sal


def abw(M: int, N: int, Kb: int, Ks: int, g: int, s: int) -> float:
    """Average bit-width ABW = S_total / (M N) (App. C.2)."""
    return storage_bits(M, N, Kb, Ks, g, s) / (M * N)


def smem_bytes(B_tile: int, Kb: int, K_tile: int, mu: int, M_tile: int) -> int:
    """Per-block shared memory of the paper's kernel (App. E.2): S_LUT = B_tile Kb (K_tile/mu) 2^mu sizeof(float),
    S_acc = B_tile Kb M_tile sizeof(float)."""
    return B_tile * Kb * (K_tile // mu) * (2 ** mu) * 4 + B_tile * Kb * M_tile * 4


def effective_tflops(M: int, N: int, N_sal: int, latency_s: float, B: int = 1) -> float:
    """Effective TFLOPS = 2 M (N + N_sal) / latency (App. E.3); multiplied by B for a batch of B."""
    return 2.0 * B * M * (N + N_sal) / latency_s / 1e12
