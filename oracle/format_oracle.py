"""Independent implementation of the packed device format, for bit-exact checks of ``fluxbin_pack``.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``). Written from the format's definition in ``include/fluxbin.h``
without any code from the library.

The format stores a "virtual" sign matrix whose columns are the global bases' columns followed by the salient bases'
VCM dense columns (Sec. 3.2, Def. VCM, Eqs. 12-13: the salient columns are remapped into a dense block so that one
kernel serves both terms). Columns are grouped in chunks of 128; every chunk of a row is 16 bytes.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .fluxbin_oracle import sign_bits

CHUNK = 128
MAGIC = 0x42584C46
VERSION = 2


def derived(spec) -> Dict[str, int]:
    """Derived sizes of the packed format.

    A chunk's row scales are "coarse" (one plane of one scale per row, shared by every chunk of the same scale group)
    when its group size is at least 128 columns or covers the whole extent, else "fine": 128 // g scales per row and
    chunk (Gcg for the global chunks, Gcs for the salient ones). When the two kinds differ and the global chunk count
    is odd, one inert chunk separates them, so that no pair of chunks (super-chunk) mixes the two layouts."""
    M, N, Kb, Ks, S = spec.M, spec.N, spec.Kb, spec.Ks, spec.S
    sal = S > 0 and Ks > 0
    Npad = -(-N // CHUNK) * CHUNK
    Sv = (-(-S // CHUNK) * CHUNK) if sal else 0
    ncg, ncs = Npad // CHUNK, Sv // CHUNK

    def per_chunk(g, extent):
        return CHUNK // g if (g < CHUNK and g < extent) else 1

    Gcg = per_chunk(spec.g_r, N)
    Gcs = per_chunk(spec.g_s, S) if sal else 1
    ngcp = Kb * ncg + (1 if (sal and Gcg != Gcs and (Kb * ncg) % 2 == 1) else 0)
    NC = ngcp + Ks * ncs
    NSC = -(-NC // 2)
    NCP = 2 * NSC
    Gr = -(-N // spec.g_r)
    Gs = (-(-S // spec.g_s)) if sal else 0
    Pg = Kb * Gr if Gcg == 1 else Kb * ncg * Gcg
    Ps = (Ks * Gs if Gcs == 1 else Ks * ncs * Gcs) if sal else 0
    return dict(Npad=Npad, Sv=Sv, ncg=ncg, ncs=ncs, NC=NC, NSC=NSC, NCP=NCP, V=CHUNK * NCP,
                Mp=-(-M // 64) * 64, Gr=Gr, Gs=Gs, NRP=Pg + Ps, Gcg=Gcg, Gcs=Gcs, ngcp=ngcp,
                nfc=ngcp if sal else NCP, Pg=Pg)


def chunk_G(spec, c: int) -> int:
    """Row scales per row of chunk c: the salient layout from the first salient chunk on (pad chunks included)."""
    d = derived(spec)
    return d["Gcg"] if c < d["nfc"] else d["Gcs"]


def chunk_info(spec, c: int):
    """(kind, base k, first local column, first row-scale plane) of chunk c; kind is 'g', 's' or 'pad'. A pad chunk
    (the separator, or the last chunk of an odd count) uses the planes of the chunk before it."""
    d = derived(spec)
    if c < spec.Kb * d["ncg"]:
        k, lc = divmod(c, d["ncg"])
        plane = k * d["Gr"] + (lc * CHUNK) // spec.g_r if d["Gcg"] == 1 else (k * d["ncg"] + lc) * d["Gcg"]
        return "g", k, lc * CHUNK, plane
    c2 = c - d["ngcp"]
    if c >= d["ngcp"] and c2 < spec.Ks * d["ncs"]:
        k, lc = divmod(c2, d["ncs"])
        if d["Gcs"] == 1:
            plane = d["Pg"] + k * d["Gs"] + (lc * CHUNK) // spec.g_s
        else:
            plane = d["Pg"] + (k * d["ncs"] + lc) * d["Gcs"]
        return "s", k, lc * CHUNK, plane
    return "pad", 0, 0, chunk_info(spec, c - 1)[3]


def position_subvector(q: int, i: int, spc: int, G: int) -> int:
    """Sub-vector held at position q of row i's entry of a chunk with G scale groups (spc positions): with n = spc / G
    positions per group, position block q // n holds group (q // n + i // n) mod G and, inside it, sub-vector
    (q mod n + i) mod n of that group."""
    n = spc // G
    return ((q // n + i // n) % G) * n + ((q % n + i) % n)


def virtual_columns(L) -> Dict[str, np.ndarray]:
    """Per virtual column: fp16 column scale (0 where no source), activation index (0xFFFF where no source); per
    chunk: row-scale plane."""
    s = L.spec
    d = derived(s)
    colscale = np.zeros(d["V"], dtype=np.uint16)
    xidx = np.full(d["V"], 0xFFFF, dtype=np.uint16)
    plane = np.zeros(d["NCP"], dtype=np.int32)
    for c in range(d["NCP"]):
        kind, k, col0, rp = chunk_info(s, c)
        plane[c] = rp
        for r in range(CHUNK):
            v = c * CHUNK + r
            if kind == "g" and col0 + r < s.N:
                j = col0 + r
                colscale[v] = L.alpha_c[k, j]
                xidx[v] = j
            elif kind == "s" and col0 + r < s.S:
                j = int(L.sal_idx[col0 + r])
                colscale[v] = L.alpha_sc[k, j]
                xidx[v] = j
    return {"colscale": colscale, "xidx": xidx, "chunk_plane": plane}


def virtual_bits(L, rows: Sequence[int]) -> np.ndarray:
    """Virtual sign bits [len(rows), V] (0/1) for the listed rows; zero where a column has no source or row >= M."""
    s = L.spec
    d = derived(s)
    rows = np.asarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, d["V"]), dtype=np.uint8)
    valid = rows < s.M
    rv = rows[valid]
    gbits = sign_bits(L.signs[:, rv], s.N) if rv.size else None
    sbits = sign_bits(L.sal_signs[:, rv], s.N) if (rv.size and s.Ks > 0) else None
    for c in range(d["NCP"]):
        kind, k, col0, _ = chunk_info(s, c)
        if kind == "g":
            n = min(CHUNK, s.N - col0)
            out[valid, c * CHUNK:c * CHUNK + n] = gbits[k][:, col0:col0 + n]
        elif kind == "s":
            n = min(CHUNK, s.S - col0)
            idx = np.asarray(L.sal_idx[col0:col0 + n], dtype=np.int64)
            out[valid, c * CHUNK:c * CHUNK + n] = sbits[k][:, idx]
    return out


def device_signs(L, rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Device sign section restricted to ``rows``: uint8 [NSC, 2, len(rows), 16].

    mu = 8: slot h of super-chunk sc for row i holds chunk 2 sc + (h xor [i mod 32 >= 16]); its byte q is the chunk's
    sub-vector byte u = position_subvector(q, i, 16, G) (G = 1: (q + i) mod 16), where sub-vector byte u packs columns
    8u..8u+7 of the chunk, LSB first.
    mu = 4: slot h holds chunk 2 sc + h; its nibble q (byte q // 2, low nibble first) is the chunk's sub-vector nibble
    u = position_subvector(q, i, 32, G), packing columns 4u..4u+3, LSB first."""
    s = L.spec
    d = derived(s)
    if rows is None:
        rows = np.arange(d["Mp"])
    rows = np.asarray(rows, dtype=np.int64)
    vb = virtual_bits(L, rows).astype(np.int64).reshape(rows.size, d["NCP"], CHUNK)
    out = np.zeros((d["NSC"], 2, rows.size, 16), dtype=np.uint8)
    if s.mu == 8:
        sub = (vb.reshape(rows.size, d["NCP"], 16, 8) << np.arange(8)).sum(-1)      # [R, NCP, 16]
        hb = ((rows % 32) >= 16).astype(np.int64)
        for sc in range(d["NSC"]):
            for h in range(2):
                c = 2 * sc + (h ^ hb)                                                  # per row
                G = np.array([chunk_G(s, int(cc)) for cc in c], dtype=np.int64)
                for q in range(16):
                    u = position_subvector(q, rows, 16, G)
                    out[sc, h, :, q] = sub[np.arange(rows.size), c, u]
    elif s.mu == 4:
        sub = (vb.reshape(rows.size, d["NCP"], 32, 4) << np.arange(4)).sum(-1)      # [R, NCP, 32]
        for sc in range(d["NSC"]):
            for h in range(2):
                c = 2 * sc + h
                G = chunk_G(s, c)
                for q in range(32):
                    u = position_subvector(q, rows, 32, G)
                    nib = sub[np.arange(rows.size), c, u]
                    out[sc, h, :, q // 2] |= (nib << (4 * (q % 2))).astype(np.uint8)
    else:
        raise ValueError("mu must be 4 or 8")
    return out


def device_rscale(L) -> np.ndarray:
    """Row-scale section: uint16 [NRP, Mp]. Coarse layout: plane k*Gr + grp holds alpha_r^(k)[:, grp] (salient: plane
    Pg + k*Gs + grp holds alpha_sr^(k)[:, grp]). Fine layout: chunk lc of base k owns the G planes starting at
    (k*nc + lc)*G (salient: after Pg), read as [Mp][G]: slot b of row i is the scale of the chunk's group
    (b + i // n) mod G, n = (128 / mu) / G, i.e. of the sub-vectors at positions b*n .. b*n + n - 1 of the row's entry.
    Groups past the last one, and rows >= M, are zero."""
    s = L.spec
    d = derived(s)
    out = np.zeros((d["NRP"], d["Mp"]), dtype=np.uint16)
    flat = out.reshape(-1)
    spc = CHUNK // s.mu

    def fine(base_plane, alpha, ngroups, nc, G, K):
        n = spc // G
        for k in range(K):
            for lc in range(nc):
                blk0 = (base_plane + (k * nc + lc) * G) * d["Mp"]
                for i in range(s.M):
                    for b in range(G):
                        grp = lc * G + (b + i // n) % G
                        if grp < ngroups:
                            flat[blk0 + i * G + b] = alpha[k, i, grp]

    if d["Gcg"] == 1:
        for k in range(s.Kb):
            for g in range(d["Gr"]):
                out[k * d["Gr"] + g, :s.M] = L.alpha_r[k, :, g]
    else:
        fine(0, L.alpha_r, d["Gr"], d["ncg"], d["Gcg"], s.Kb)
    if d["Gs"]:
        if d["Gcs"] == 1:
            for k in range(s.Ks):
                for g in range(d["Gs"]):
                    out[d["Pg"] + k * d["Gs"] + g, :s.M] = L.alpha_sr[k, :, g]
        else:
            fine(d["Pg"], L.alpha_sr, d["Gs"], d["ncs"], d["Gcs"], s.Ks)
    return out


def device_sal_idx(L) -> np.ndarray:
    """Salient index section: uint16 [max(S, 1)] (16-bit indices as in App. C.2); a lone 0 when S = 0."""
    s = L.spec
    out = np.zeros(max(s.S, 1), dtype=np.uint16)
    out[:s.S] = np.asarray(L.sal_idx, dtype=np.int64)
    return out


def undo_device_signs(dev: np.ndarray, spec, rows: Sequence[int]) -> np.ndarray:
    """Inverse of ``device_signs``: uint8 [NSC, 2, R, 16] -> virtual bits [R, V]. Written as a scatter, independently
    of the gather above, to pin that the layout is a bijection."""
    d = derived(spec)
    rows = np.asarray(rows, dtype=np.int64)
    vb = np.zeros((rows.size, d["NCP"], CHUNK), dtype=np.uint8)
    for ri, i in enumerate(rows):
        for sc in range(d["NSC"]):
            for h in range(2):
                if spec.mu == 8:
                    c = 2 * sc + (h ^ int((i % 32) >= 16))
                    for q in range(16):
                        u = position_subvector(q, int(i), 16, chunk_G(spec, c))
                        byte = int(dev[sc, h, ri, q])
                        for n in range(8):
                            vb[ri, c, 8 * u + n] = (byte >> n) & 1
                else:
                    c = 2 * sc + h
                    for q in range(32):
                        u = position_subvector(q, int(i), 32, chunk_G(spec, c))
                        nib = (int(dev[sc, h, ri, q // 2]) >> (4 * (q % 2))) & 15
                        for n in range(4):
                            vb[ri, c, 4 * u + n] = (nib >> n) & 1
    return vb.reshape(rows.size, d["V"])


def packed_bytes(spec) -> Dict[str, int]:
    """Section sizes, offsets (each a multiple of 256) and the total size of the packed buffer."""
    d = derived(spec)
    sizes = [
        ("header", 256),
        ("signs", d["NSC"] * 2 * d["Mp"] * 16),
        ("rscale", d["NRP"] * d["Mp"] * 2),
        ("colscale", d["V"] * 2),
        ("xidx", d["V"] * 2),
        ("chunk_plane", d["NCP"] * 4),
        ("sal_idx", max(spec.S, 1) * 2),
    ]
    off = 0
    out = {}
    for name, sz in sizes:
        out["off_" + name] = off
        out["size_" + name] = sz
        off += -(-sz // 256) * 256
    out["total"] = off
    return out
