// Packing kernels of libfluxbin: canonical planes -> device format (relayout of the sign planes, VCM extraction of
// the salient columns, gather of their column scales), plus the layout-decoding kernels used by tests.
//
// VCM (Sec. 3.2, Def. VCM, Eqs. 12-13): the salient columns of each salient base are copied into a dense block of
// virtual columns (dense column t <- input column I_sal[t]) and their column scales are gathered once here, so the
// GEMV kernels read the salient refinement exactly like the global bases.
#include <hip/hip_runtime.h>

#include "fluxbin_internal.h"

namespace fluxbin {

struct PackArgs {
  const uint32_t* signs;
  const uint32_t* sal_signs;
  const int32_t* sal_idx;
  const uint16_t* alpha_r;
  const uint16_t* alpha_c;
  const uint16_t* alpha_sr;
  const uint16_t* alpha_sc;
  uint8_t* base;
  int64_t M, N, W, g_r, S, g_s;
  int32_t Kb, Ks, mu, pad0;
  int64_t Npad, ncg, Sv, ncs, NC, NSC, NCP, V, Mp, Gr, Gs, NRP;
  int64_t Gcg, Gcs, ngcp, nfc, Pg;
  uint64_t off_signs, off_rscale, off_colscale, off_xidx, off_chunk_plane, off_sal_idx;
};

struct HeaderWords {
  uint32_t w[64];
};

// Kind of chunk c: 0 global, 1 salient, 2 pad (the separator after the global chunks, or the last chunk of an odd
// count); base k and the first local column.
__device__ inline int chunk_kind(const PackArgs& a, int64_t c, int64_t* k, int64_t* col0) {
  if (c < a.Kb * a.ncg) {
    *k = c / a.ncg;
    *col0 = (c % a.ncg) * kChunk;
    return 0;
  }
  if (c < a.ngcp) {
    *k = 0;
    *col0 = 0;
    return 2;
  }
  const int64_t c2 = c - a.ngcp;
  if (c2 < a.Ks * a.ncs) {
    *k = c2 / a.ncs;
    *col0 = (c2 % a.ncs) * kChunk;
    return 1;
  }
  *k = 0;
  *col0 = 0;
  return 2;
}

// Row scales per chunk c and row (1: one plane; G > 1: a block of G scales per row), by the chunk's scale layout.
__device__ inline int64_t chunk_G(const PackArgs& a, int64_t c) { return c < a.nfc ? a.Gcg : a.Gcs; }

// Sub-vector held at position q of row i's 16-byte entry of a chunk with G scale groups (spc = 128/mu positions,
// n = spc/G per group): the groups are rotated by floor(i/n) and the positions within a group by i, so that any
// spc consecutive rows read spc different sub-vectors at every position (G = 1: (q + i) mod spc).
__device__ inline int sub_at(int q, int64_t i, int spc, int G) {
  const int n = spc / G;
  const int blk = int(((q / n) + (i / n)) % G);
  const int w = int(((q % n) + i) % n);
  return blk * n + w;
}

// Inverse of sub_at: the position of sub-vector u.
__device__ inline int pos_of(int u, int64_t i, int spc, int G) {
  const int n = spc / G;
  const int blk = int((((u / n) - (i / n)) % G + G) % G);
  const int w = int((((u % n) - i) % n + n) % n);
  return blk * n + w;
}

// The 128 virtual sign bits of chunk c for row i (bit r of the result <-> virtual column 128 c + r).
__device__ inline void chunk_bits(const PackArgs& a, int64_t c, int64_t i, uint32_t out[4]) {
  out[0] = out[1] = out[2] = out[3] = 0u;
  if (i >= a.M) return;
  int64_t k, col0;
  const int kind = chunk_kind(a, c, &k, &col0);
  if (kind == 0) {
    const uint32_t* row = a.signs + (k * a.M + i) * a.W;
    for (int m = 0; m < 4; ++m) {
      const int64_t j0 = col0 + 32 * m;
      if (j0 >= a.N) break;
      uint32_t word = row[j0 / 32];
      const int64_t valid = a.N - j0;
      if (valid < 32) word &= (1u << valid) - 1u;
      out[m] = word;
    }
  } else if (kind == 1) {
    const uint32_t* row = a.sal_signs + (k * a.M + i) * a.W;
    for (int r = 0; r < kChunk; ++r) {
      const int64_t t = col0 + r;
      if (t >= a.S) break;
      const int64_t j = a.sal_idx[t];
      const uint32_t bit = (row[j >> 5] >> (j & 31)) & 1u;
      out[r >> 5] |= bit << (r & 31);
    }
  }
}

// One thread per 16-byte entry (super-chunk sc, slot h, row i < Mp).
__global__ void k_pack_signs(PackArgs a) {
  const int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  const int64_t n = a.NSC * 2 * a.Mp;
  if (e >= n) return;
  const int64_t i = e % a.Mp;
  const int64_t sh = e / a.Mp;
  const int64_t sc = sh >> 1;
  const int64_t h = sh & 1;
  uint32_t bits[4];
  uint32_t o[4] = {0u, 0u, 0u, 0u};
  if (a.mu == 8) {
    const int64_t c = 2 * sc + (h ^ ((i & 31) >= 16 ? 1 : 0));
    chunk_bits(a, c, i, bits);
    const int G = int(chunk_G(a, c));
    for (int q = 0; q < 16; ++q) {
      const int u = sub_at(q, i, 16, G);
      const uint32_t byte = (bits[u >> 2] >> (8 * (u & 3))) & 0xFFu;
      o[q >> 2] |= byte << (8 * (q & 3));
    }
  } else {
    const int64_t c = 2 * sc + h;
    chunk_bits(a, c, i, bits);
    const int G = int(chunk_G(a, c));
    for (int q = 0; q < 32; ++q) {
      const int u = sub_at(q, i, 32, G);
      const uint32_t nib = (bits[u >> 3] >> (4 * (u & 7))) & 0xFu;
      o[q >> 3] |= nib << (4 * (q & 7));
    }
  }
  uint4* dst = reinterpret_cast<uint4*>(a.base + a.off_signs) + e;
  *dst = make_uint4(o[0], o[1], o[2], o[3]);
}

// One thread per (row-scale plane, row < Mp). Coarse planes hold one scale per row; a fine chunk's block of G planes
// holds, for each row, G consecutive scales: slot b is the scale of the chunk's group (b + floor(i/n)) mod G (n = spc/G
// sub-vectors per group), i.e. the group read at positions b*n .. b*n+n-1 of the row's rotated entry.
__global__ void k_pack_rscale(PackArgs a) {
  const int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (e >= a.NRP * a.Mp) return;
  const bool salient = e >= a.Pg * a.Mp;
  const int64_t G = salient ? a.Gcs : a.Gcg;
  const int64_t e2 = salient ? e - a.Pg * a.Mp : e;
  uint16_t v = 0;
  if (G == 1) {
    const int64_t i = e2 % a.Mp;
    const int64_t plane = e2 / a.Mp;
    if (i < a.M) {
      if (!salient) {
        const int64_t k = plane / a.Gr, g = plane % a.Gr;
        v = a.alpha_r[(k * a.M + i) * a.Gr + g];
      } else {
        const int64_t k = plane / a.Gs, g = plane % a.Gs;
        v = a.alpha_sr[(k * a.M + i) * a.Gs + g];
      }
    }
  } else {
    const int64_t blk = e2 / (a.Mp * G);                 // (base, chunk within the base)
    const int64_t i = (e2 % (a.Mp * G)) / G;
    const int64_t b = e2 % G;
    const int64_t nc = salient ? a.ncs : a.ncg;
    const int64_t k = blk / nc, lc = blk % nc;
    const int64_t n = (kChunk / a.mu) / G;
    const int64_t grp = lc * G + (b + i / n) % G;
    if (i < a.M) {
      if (!salient && grp < a.Gr) v = a.alpha_r[(k * a.M + i) * a.Gr + grp];
      if (salient && grp < a.Gs) v = a.alpha_sr[(k * a.M + i) * a.Gs + grp];
    }
  }
  reinterpret_cast<uint16_t*>(a.base + a.off_rscale)[e] = v;
}

// One thread per virtual column; the first NCP threads also write the chunk's row-scale plane, the first max(S,1)
// threads the 16-bit salient indices.
__global__ void k_pack_columns(PackArgs a) {
  const int64_t v = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (v < a.V) {
    const int64_t c = v / kChunk;
    const int64_t r = v % kChunk;
    int64_t k, col0;
    const int kind = chunk_kind(a, c, &k, &col0);
    uint16_t cs = 0, xi = 0xFFFFu;
    if (kind == 0 && col0 + r < a.N) {
      const int64_t j = col0 + r;
      cs = a.alpha_c[k * a.N + j];
      xi = uint16_t(j);
    } else if (kind == 1 && col0 + r < a.S) {
      const int64_t j = a.sal_idx[col0 + r];
      cs = a.alpha_sc[k * a.N + j];
      xi = uint16_t(j);
    }
    reinterpret_cast<uint16_t*>(a.base + a.off_colscale)[v] = cs;
    reinterpret_cast<uint16_t*>(a.base + a.off_xidx)[v] = xi;
  }
  if (v < a.NCP) {
    // first row-scale plane of chunk v; a pad chunk uses the planes of the chunk before it (its signs and column
    // scales are zero, so any finite scale gives it exactly zero)
    int64_t c = v;
    int64_t k, col0;
    int kind = chunk_kind(a, c, &k, &col0);
    while (kind == 2 && c > 0) kind = chunk_kind(a, --c, &k, &col0);
    int64_t plane = 0;
    if (kind == 0) plane = a.Gcg == 1 ? k * a.Gr + col0 / a.g_r : (k * a.ncg + col0 / kChunk) * a.Gcg;
    if (kind == 1) plane = a.Pg + (a.Gcs == 1 ? k * a.Gs + col0 / a.g_s : (k * a.ncs + col0 / kChunk) * a.Gcs);
    reinterpret_cast<int32_t*>(a.base + a.off_chunk_plane)[v] = int32_t(plane);
  }
  const int64_t ns = a.S > 1 ? a.S : 1;
  if (v < ns) {
    reinterpret_cast<uint16_t*>(a.base + a.off_sal_idx)[v] = (v < a.S) ? uint16_t(a.sal_idx[v]) : uint16_t(0);
  }
}

__global__ void k_write_header(HeaderWords h, uint32_t* dst) {
  const int t = threadIdx.x;
  if (t < 64) dst[t] = h.w[t];
}

// Reads one virtual sign bit (chunk c, column r of the chunk, row i) back from the device layout.
__device__ inline uint32_t device_bit(const PackArgs& a, const uint8_t* signs, int64_t c, int r, int64_t i) {
  const int64_t Mp = a.Mp;
  const int mu = a.mu;
  const int G = int(chunk_G(a, c));
  const int64_t sc = c >> 1;
  if (mu == 8) {
    const int64_t h = (c & 1) ^ ((i & 31) >= 16 ? 1 : 0);
    const int u = r >> 3, n = r & 7;
    const int q = pos_of(u, i, 16, G);
    const uint8_t byte = signs[((sc * 2 + h) * Mp + i) * 16 + q];
    return (byte >> n) & 1u;
  }
  const int64_t h = c & 1;
  const int u = r >> 2, n = r & 3;
  const int q = pos_of(u, i, 32, G);
  const uint8_t byte = signs[((sc * 2 + h) * Mp + i) * 16 + (q >> 1)];
  return (byte >> (4 * (q & 1) + n)) & 1u;
}

// One thread per output word: global planes [Kb][M][W] then dense salient planes [Ks][M][ceil(S/32)].
__global__ void k_unpack(PackArgs a, uint32_t* d_signs, uint32_t* d_dense) {
  const int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  const uint8_t* signs = a.base + a.off_signs;
  const int64_t ng = a.Kb * a.M * a.W;
  const int64_t Ws = (a.S + 31) / 32;
  const int64_t ns = (d_dense && a.Ks > 0 && a.S > 0) ? a.Ks * a.M * Ws : 0;
  if (e < ng) {
    const int64_t w = e % a.W, i = (e / a.W) % a.M, k = e / (a.W * a.M);
    uint32_t word = 0;
    for (int b = 0; b < 32; ++b) {
      const int64_t j = 32 * w + b;
      if (j >= a.N) break;
      const int64_t vcol = k * a.Npad + j;
      word |= device_bit(a, signs, vcol / kChunk, int(vcol % kChunk), i) << b;
    }
    d_signs[e] = word;
  } else if (e < ng + ns) {
    const int64_t f = e - ng;
    const int64_t w = f % Ws, i = (f / Ws) % a.M, k = f / (Ws * a.M);
    uint32_t word = 0;
    for (int b = 0; b < 32; ++b) {
      const int64_t t = 32 * w + b;
      if (t >= a.S) break;
      const int64_t vcol = a.ngcp * kChunk + k * a.Sv + t;
      word |= device_bit(a, signs, vcol / kChunk, int(vcol % kChunk), i) << b;
    }
    d_dense[f] = word;
  }
}

// Pattern read at step q from the 16-byte entry of a row (the same byte/nibble selection the GEMV kernels make).
__device__ inline uint32_t pattern_at(const uint4& e, int q, int mu) {
  const uint32_t w[4] = {e.x, e.y, e.z, e.w};
  if (mu == 8) return (w[q >> 2] >> (8 * (q & 3))) & 0xFFu;
  return (w[q >> 3] >> (4 * (q & 7))) & 0xFu;
}

// One thread per (chunk c, row i < M, sub-vector u): the LUT index the kernels read for that sub-vector.
__global__ void k_debug_indices(PackArgs a, uint8_t* d_p) {
  const int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  const int per = kChunk / a.mu;
  if (e >= a.NCP * a.M * per) return;
  const int u = int(e % per);
  const int64_t i = (e / per) % a.M;
  const int64_t c = e / (per * a.M);
  const int64_t sc = c >> 1;
  int64_t h;
  int q;
  const int G = int(chunk_G(a, c));
  if (a.mu == 8) {
    h = (c & 1) ^ ((i & 31) >= 16 ? 1 : 0);
    q = pos_of(u, i, 16, G);
  } else {
    h = c & 1;
    q = pos_of(u, i, 32, G);
  }
  const uint4 entry = reinterpret_cast<const uint4*>(a.base + a.off_signs)[(sc * 2 + h) * a.Mp + i];
  d_p[e] = uint8_t(pattern_at(entry, q, a.mu));
}

__global__ void k_fill_zero(uint32_t* d, int64_t n) {
  const int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x;
  if (e < n) d[e] = 0u;
}

static PackArgs make_args(const fluxbin_layer& L) {
  PackArgs a{};
  const fluxbin_shape& s = L.shape;
  const Derived d = derive(s);
  a.base = static_cast<uint8_t*>(L.d_base);
  a.M = s.M;
  a.N = s.N;
  a.W = (s.N + 31) / 32;
  a.g_r = s.g_r;
  a.S = s.S;
  a.g_s = s.g_s;
  a.Kb = s.Kb;
  a.Ks = s.Ks;
  a.mu = s.mu;
  a.Npad = d.Npad;
  a.ncg = d.ncg;
  a.Sv = d.Sv;
  a.ncs = d.ncs;
  a.NC = d.NC;
  a.NSC = d.NSC;
  a.NCP = d.NCP;
  a.V = d.V;
  a.Mp = d.Mp;
  a.Gr = d.Gr;
  a.Gs = d.Gs;
  a.NRP = d.NRP;
  a.Gcg = d.Gcg;
  a.Gcs = d.Gcs;
  a.ngcp = d.ngcp;
  a.nfc = d.nfc;
  a.Pg = d.Pg;
  a.off_signs = L.off_signs;
  a.off_rscale = L.off_rscale;
  a.off_colscale = L.off_colscale;
  a.off_xidx = L.off_xidx;
  a.off_chunk_plane = L.off_chunk_plane;
  a.off_sal_idx = L.off_sal_idx;
  return a;
}

static unsigned grid_for(int64_t n, int threads) { return unsigned((n + threads - 1) / threads); }

fluxbin_status launch_pack(const fluxbin_layer& L, const fluxbin_weights& w, const int32_t* d_sal_idx,
                           hipStream_t stream) {
  PackArgs a = make_args(L);
  a.signs = w.signs;
  a.sal_signs = w.sal_signs;
  a.sal_idx = d_sal_idx;
  a.alpha_r = w.alpha_r;
  a.alpha_c = w.alpha_c;
  a.alpha_sr = w.alpha_sr;
  a.alpha_sc = w.alpha_sc;
  const Derived d = derive(L.shape);
  const Offsets o = offsets(L.shape, d);
  Header h{};
  h.magic = kMagic;
  h.version = FLUXBIN_FORMAT_VERSION;
  h.shape = L.shape;
  h.Npad = d.Npad;
  h.Sv = d.Sv;
  h.NC = d.NC;
  h.NSC = d.NSC;
  h.Mp = d.Mp;
  h.Gr = d.Gr;
  h.Gs = d.Gs;
  h.NRP = d.NRP;
  h.off_signs = o.signs;
  h.off_rscale = o.rscale;
  h.off_colscale = o.colscale;
  h.off_xidx = o.xidx;
  h.off_chunk_plane = o.chunk_plane;
  h.off_sal_idx = o.sal_idx;
  h.total = o.total;
  HeaderWords hw;
  static_assert(sizeof(hw) == sizeof(h), "header size");
  __builtin_memcpy(&hw, &h, sizeof(h));

  const int T = 256;
  hipLaunchKernelGGL(k_write_header, dim3(1), dim3(64), 0, stream, hw, static_cast<uint32_t*>(L.d_base));
  const int64_t n_sig = d.NSC * 2 * d.Mp;
  hipLaunchKernelGGL(k_pack_signs, dim3(grid_for(n_sig, T)), dim3(T), 0, stream, a);
  if (d.NRP * d.Mp > 0) hipLaunchKernelGGL(k_pack_rscale, dim3(grid_for(d.NRP * d.Mp, T)), dim3(T), 0, stream, a);
  int64_t n_col = d.V;
  if (L.shape.S > n_col) n_col = L.shape.S;
  hipLaunchKernelGGL(k_pack_columns, dim3(grid_for(n_col, T)), dim3(T), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the packing kernels");
  return FLUXBIN_OK;
}

fluxbin_status launch_unpack(const fluxbin_layer& L, uint32_t* d_signs, uint32_t* d_dense, hipStream_t stream) {
  PackArgs a = make_args(L);
  const int64_t ng = a.Kb * a.M * a.W;
  const int64_t ns = (d_dense && a.Ks > 0 && a.S > 0) ? a.Ks * a.M * ((a.S + 31) / 32) : 0;
  const int T = 256;
  hipLaunchKernelGGL(k_unpack, dim3(grid_for(ng + ns, T)), dim3(T), 0, stream, a, d_signs, d_dense);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the unpack kernel");
  return FLUXBIN_OK;
}

fluxbin_status launch_debug_indices(const fluxbin_layer& L, uint8_t* d_p, hipStream_t stream) {
  PackArgs a = make_args(L);
  const int64_t n = a.NCP * a.M * (kChunk / a.mu);
  const int T = 256;
  hipLaunchKernelGGL(k_debug_indices, dim3(grid_for(n, T)), dim3(T), 0, stream, a, d_p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the debug-indices kernel");
  return FLUXBIN_OK;
}

fluxbin_status launch_fill_zero(void* d, size_t bytes, hipStream_t stream) {
  const int64_t n = int64_t(bytes / 4);
  const int T = 256;
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for(n, T)), dim3(T), 0, stream, static_cast<uint32_t*>(d), n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the fill kernel");
  return FLUXBIN_OK;
}

}  // namespace fluxbin
