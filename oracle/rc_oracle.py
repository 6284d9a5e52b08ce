"""Oracle of FluxBin's weight decomposition: plain, slow, fp64 CPU reference.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this module. It shares no code with the HIP path (``paper_2608_15602_amd/``) and never imports it.

What it follows (FluxBin, arXiv 2608.15602):
  * Def. Row-Column Binary Decomposition (Sec. 3.1): W^(k) = (alpha_r^(k) alpha_c^(k)^T) * B^(k), B in {-1, +1},
    one row scale per group of columns;
  * Prop. 3.2 (Optimal Scaling Factors): with B and one scale vector fixed, each entry of the other vector is the
    weighted least-squares solution  sum(c * B * W) / (sum((c * B)^2) + eps);
  * Prop. 3.3 (Optimal Binary Base Assignment): with all scales fixed, each element's signs (b_1..b_K) minimize
    |W_ij - sum_k M_ij^(k) b_k| over the 2^K combinations, searched exhaustively;
  * Def. Hessian-based Column Saliency (Sec. 3.1): S_j = sum_i W_ij^2 / [H^-1]_jj^2, and per group of g columns the s
    columns of largest total saliency;
  * the RC_Decomp sub-routine (App. algorithm "FluxBin Sub-routines"): greedy residual initialization of every base,
    then T rounds of (row and column scale updates for each base, joint sign search, signs times the mask), and the
    hybrid procedure (App. algorithm "FluxBin-Hybrid"): per block of g columns saliency search, global bases, salient
    refinement of the residual on the salient columns.

Readings where the paper is silent:
  * greedy initialization of base k from the residual R: B = sign(R) on the mask (sign(0) = +1), 0 off it; the column
    scale starts at 1, then the row scale and the column scale take one least-squares update each (Prop. 3.2, in that
    order); R loses the base's contribution;
  * in the alternating rounds the target of base k is X * mask minus the other bases' current contributions; bases
    are visited in order k = 1..K, row scale before column scale, each update seeing the latest values;
  * ties in the sign search keep the first combination in the order c = 0..2^K-1, where bit k of c set means b_k = +1;
  * one row scale per (row, block of g columns): the blocks are decomposed independently (with a diagonal inverse
    Hessian the GPTQ error compensation between blocks is exactly zero, the synthetic setting used here);
  * the salient refinement follows the hybrid procedure block by block: within each block of g columns, RC_Decomp of
    the block's residual (after its global bases) on the block's salient mask, so every salient base has one row
    scale per (row, block), the 16*M*N/g term of the storage analysis (App. C.2); in the packed format's dense salient
    columns that is one scale per s columns (g_s = s);
  * the top-s selection orders columns by decreasing saliency, equal scores by increasing column index;
  * eps = 1e-12 (the paper names a stability constant without a value).
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

EPS = 1e-12


def row_update(target: np.ndarray, B: np.ndarray, alpha_c: np.ndarray, eps: float = EPS) -> np.ndarray:
    """Prop. 3.2, row form: alpha_r[i] = sum_j (c_j B_ij) T_ij / (sum_j (c_j B_ij)^2 + eps) for one block."""
    cb = alpha_c[None, :] * B
    return (cb * target).sum(axis=1) / ((cb * cb).sum(axis=1) + eps)


def col_update(target: np.ndarray, B: np.ndarray, alpha_r_cols: np.ndarray, eps: float = EPS) -> np.ndarray:
    """Prop. 3.2, column form: alpha_c[j] = sum_i (r_ij B_ij) T_ij / (sum_i (r_ij B_ij)^2 + eps), where r_ij is the row
    scale of row i in column j's block (alpha_r_cols holds it per element)."""
    rb = alpha_r_cols * B
    return (rb * target).sum(axis=0) / ((rb * rb).sum(axis=0) + eps)


def sign_search(X: np.ndarray, mags: List[np.ndarray]) -> np.ndarray:
    """Prop. 3.3: per element the signs b in {-1,+1}^K minimizing |X - sum_k mags[k] b_k|, by trying every combination
    c = 0..2^K-1 (bit k of c set: b_k = +1) and keeping the first minimum. Returns int8 [K, ...]."""
    K = len(mags)
    best = np.full(X.shape, np.inf)
    out = np.zeros((K,) + X.shape, dtype=np.int8)
    for c in range(1 << K):
        b = [1 if (c >> k) & 1 else -1 for k in range(K)]
        approx = np.zeros_like(X)
        for k in range(K):
            approx = approx + mags[k] * b[k]
        err = np.abs(X - approx)
        better = err < best
        best = np.where(better, err, best)
        for k in range(K):
            out[k] = np.where(better, b[k], out[k])
    return out


def _expand_rows(alpha_r: np.ndarray, g: int, N: int) -> np.ndarray:
    """[M, G] row scales -> [M, N] (each column gets the row scale of its block)."""
    return np.repeat(alpha_r, g, axis=1)[:, :N]


def reconstruct(B: np.ndarray, alpha_r: np.ndarray, alpha_c: np.ndarray, g: int) -> np.ndarray:
    """sum_k (alpha_r^(k) alpha_c^(k)^T) * B^(k) with block row scales (Def. RC decomposition)."""
    K, M, N = B.shape
    out = np.zeros((M, N))
    for k in range(K):
        out += _expand_rows(alpha_r[k], g, N) * alpha_c[k][None, :] * B[k]
    return out


def rc_decomp(X: np.ndarray, mask: np.ndarray, K: int, T: int, g: int, eps: float = EPS) -> Dict[str, np.ndarray]:
    """RC_Decomp(X, mask, K, T) on every block of g columns of X [M, N] (N need not be a multiple of g; the last block
    is shorter). mask: bool [N] (columns included). Returns B int8 [K, M, N] (0 off the mask), alpha_r [K, M, G],
    alpha_c [K, N] and the loss ||X*mask - W-hat||_F^2 after the initialization and after every round."""
    X = np.asarray(X, dtype=np.float64)
    M, N = X.shape
    G = -(-N // g)
    m = np.asarray(mask, dtype=bool)
    Xm = X * m[None, :]
    B = np.zeros((K, M, N), dtype=np.int8)
    ar = np.zeros((K, M, G))
    ac = np.zeros((K, N))

    def contribution(k):
        return _expand_rows(ar[k], g, N) * ac[k][None, :] * B[k]

    def update_scales(k, target):
        for blk in range(G):
            cols = slice(blk * g, min(N, (blk + 1) * g))
            ar[k][:, blk] = row_update(target[:, cols], B[k][:, cols].astype(np.float64), ac[k][cols], eps)
        ac[k] = col_update(target, B[k].astype(np.float64), _expand_rows(ar[k], g, N), eps)

    # greedy residual initialization
    R = Xm.copy()
    for k in range(K):
        B[k] = np.where(m[None, :], np.where(R >= 0, 1, -1), 0).astype(np.int8)
        ac[k] = 1.0
        update_scales(k, R)
        R = R - contribution(k)
    losses = [float(((Xm - reconstruct(B, ar, ac, g)) ** 2).sum())]
    # alternating optimization
    for _ in range(T):
        for k in range(K):
            target = Xm - sum(contribution(kk) for kk in range(K) if kk != k)
            update_scales(k, target)
        mags = [_expand_rows(ar[k], g, N) * ac[k][None, :] for k in range(K)]
        B = sign_search(Xm, mags)
        B = np.where(m[None, None, :], B, 0).astype(np.int8)
        losses.append(float(((Xm - reconstruct(B, ar, ac, g)) ** 2).sum()))
    return dict(B=B, alpha_r=ar, alpha_c=ac, loss=np.array(losses))


def saliency(W: np.ndarray, hinv_diag: np.ndarray) -> np.ndarray:
    """Def. Hessian-based Column Saliency: S_j = sum_i W_ij^2 / [H^-1]_jj^2."""
    W = np.asarray(W, dtype=np.float64)
    return (W * W).sum(axis=0) / (np.asarray(hinv_diag, dtype=np.float64) ** 2)


def structural_search(W: np.ndarray, hinv_diag: np.ndarray, g: int, s: int) -> np.ndarray:
    """Per block of g columns the s columns of largest saliency (decreasing score, equal scores by increasing index);
    the union over blocks, sorted (int64). A block shorter than s contributes all its columns."""
    S = saliency(W, hinv_diag)
    N = S.shape[0]
    out = []
    for b0 in range(0, N, g):
        cols = np.arange(b0, min(N, b0 + g))
        order = sorted(cols.tolist(), key=lambda j: (-S[j], j))
        out.extend(order[:s])
    return np.array(sorted(out), dtype=np.int64)


def hybrid_quantize(W: np.ndarray, hinv_diag: np.ndarray, g: int, s: int, Kb: int, Ks: int, T: int,
                    eps: float = EPS) -> Dict[str, np.ndarray]:
    """FluxBin-Hybrid (App. algorithm "FluxBin-Hybrid") with a diagonal inverse Hessian, block by block over the
    column blocks of g: (1) structural search picks the block's s salient columns; (2) RC_Decomp of the block into Kb
    global bases (all columns); (3) RC_Decomp of the block's residual into Ks salient bases on the block's mask. The
    error compensation between blocks (step 4) is zero for a diagonal inverse Hessian, so the blocks are independent.
    Returns the salient columns and, per branch, the bases of all blocks side by side: signs [K, M, N], row scales
    [K, M, ceil(N/g)] (one per row and block), column scales [K, N]."""
    W = np.asarray(W, dtype=np.float64)
    M, N = W.shape
    G = -(-N // g)
    sal_parts = []
    glob = dict(B=np.zeros((Kb, M, N), dtype=np.int8), alpha_r=np.zeros((Kb, M, G)), alpha_c=np.zeros((Kb, N)))
    salr = (dict(B=np.zeros((Ks, M, N), dtype=np.int8), alpha_r=np.zeros((Ks, M, G)), alpha_c=np.zeros((Ks, N)))
            if Ks > 0 else None)
    for blk in range(G):
        cols = slice(blk * g, min(N, (blk + 1) * g))
        Wb = W[:, cols]
        nb = Wb.shape[1]
        idx = structural_search(Wb, np.asarray(hinv_diag, dtype=np.float64)[cols], nb, s)   # step 1
        sal_parts.append(idx + blk * g)
        gb = rc_decomp(Wb, np.ones(nb, dtype=bool), Kb, T, nb, eps)                      # step 2
        glob["B"][:, :, cols] = gb["B"]
        glob["alpha_r"][:, :, blk] = gb["alpha_r"][:, :, 0]
        glob["alpha_c"][:, cols] = gb["alpha_c"]
        if Ks > 0:                                                                        # step 3
            Rb = Wb - reconstruct(gb["B"], gb["alpha_r"], gb["alpha_c"], nb)
            mb = np.zeros(nb, dtype=bool)
            mb[idx] = True
            sb = rc_decomp(Rb, mb, Ks, T, nb, eps)
            salr["B"][:, :, cols] = sb["B"]
            salr["alpha_r"][:, :, blk] = sb["alpha_r"][:, :, 0]
            salr["alpha_c"][:, cols] = sb["alpha_c"]
    return dict(sal_idx=np.concatenate(sal_parts).astype(np.int64), glob=glob, sal=salr)
