// LUT-GEMV / small-batch LUT-GEMM kernels of libfluxbin for gfx950 (CDNA4).
//
// What is computed (Sec. 3.2): y[b, i] = sum over the virtual columns of the packed format of
//   rscale[plane(c)][i] * sum_{sub-vectors s of chunk c} LUT_{b,c,s}[p(i, c, s)]
// where LUT_{b,c,s}[p] = sum_n xv[b, 128c + mu s + n] * (2 bit_n(p) - 1) is the LUT-BSF table of Eq. (14) built from
// xv = x[xidx] * colscale (column scale folded into the activation, Eq. 11; VCM gather for salient columns, Eq. 13),
// and the row scale multiplies the summed lookups of its group (Eq. 15).
//
// Work decomposition. A tile is `rows` consecutive output rows; a unit is one tile times one step of the virtual
// columns (a super-chunk of 256 columns for the batch-1 mu=8 kernel; one chunk of 128 columns times one group of batch
// rows for the generic kernel). The units are numbered tile-major and split into `blocks` contiguous, equal ranges
// (one per workgroup), so every workgroup streams the same number of sign bytes. A tile covered by several
// workgroups is reduced by the last of them to finish (a 32-bit counter per tile, no float atomics): it adds the
// partial sums in workgroup order, so the result does not depend on timing.
//
// Per unit a workgroup builds the tables of the next unit in LDS while it reads the current one (double buffer), and
// the sign words of the next unit are in flight during the current lookups.
#include <hip/hip_runtime.h>

#include "fluxbin_internal.h"

namespace fluxbin {

struct GemmArgs {
  const uint8_t* signs;
  const uint16_t* rscale;
  const uint16_t* colscale;
  const uint16_t* xidx;
  const int32_t* chunk_plane;
  const uint16_t* x;
  void* y;
  float* partials;
  uint32_t* counters;
  int64_t ldx, ldy;
  int64_t units, blocks;
  int32_t M, Mp, NSC, NCP;
  int32_t steps;   // units per tile
  int32_t B;       // batch rows actually present
  int32_t y_fp32;
  int32_t n_tiles;
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float h2f(uint16_t u) { return static_cast<float>(__builtin_bit_cast(_Float16, u)); }

__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f)); }

__device__ __forceinline__ uint4 load_stream16(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Workgroup that owns unit u when `units` units are split into `blocks` ranges [b*units/blocks, (b+1)*units/blocks).
__device__ __forceinline__ int64_t owner_of(int64_t u, int64_t units, int64_t blocks) {
  return ((u + 1) * blocks + units - 1) / units - 1;
}

__device__ __forceinline__ void store_y(const GemmArgs& a, int b, int64_t row, float v) {
  if (a.y_fp32)
    static_cast<float*>(a.y)[b * a.ldy + row] = v;
  else
    static_cast<uint16_t*>(a.y)[b * a.ldy + row] = f2h(v);
}

// End of a tile's contribution from this workgroup: store y directly when the workgroup covers the whole tile,
// otherwise publish the partial sums; the last contributor adds them in workgroup order and stores y.
// acc is [RPT][BP] (row j of this thread, batch row b).
template <int NT, int RPT, int BP>
__device__ __forceinline__ void finish_tile(const GemmArgs& a, int64_t tile, int64_t first_tile, float (&acc)[RPT][BP],
                                            int* s_flag) {
  const int t = threadIdx.x;
  const int64_t R = int64_t(NT) * RPT;
  const int64_t b_self = blockIdx.x;
  const int64_t b_first = owner_of(tile * a.steps, a.units, a.blocks);
  const int64_t b_last = owner_of((tile + 1) * a.steps - 1, a.units, a.blocks);
  if (b_first == b_last) {
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int64_t row = tile * R + t + NT * j;
      if (row < a.M) {
#pragma unroll
        for (int b = 0; b < BP; ++b)
          if (b < a.B) store_y(a, b, row, acc[j][b]);
      }
    }
    return;
  }
  // partial slot of a workgroup for a tile: 0 for its first tile, 1 for its last one
  const int slot = (tile == first_tile) ? 0 : 1;
  float* mine = a.partials + ((b_self * 2 + slot) * BP) * R;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
#pragma unroll
    for (int b = 0; b < BP; ++b) mine[b * R + t + NT * j] = acc[j][b];
  }
  __threadfence();
  __syncthreads();
  if (t == 0) {
    const uint32_t prev = atomicAdd(a.counters + tile, 1u);
    *s_flag = (prev == uint32_t(b_last - b_first)) ? 1 : 0;
  }
  __syncthreads();
  if (*s_flag) {
    __threadfence();
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int64_t r = t + NT * j;
      const int64_t row = tile * R + r;
      float sum[BP];
#pragma unroll
      for (int b = 0; b < BP; ++b) sum[b] = 0.f;
      for (int64_t bb = b_first; bb <= b_last; ++bb) {
        const int64_t first_of_bb = (bb * a.units / a.blocks) / a.steps;
        const int sl = (tile == first_of_bb) ? 0 : 1;
        const float* src = a.partials + ((bb * 2 + sl) * BP) * R;
#pragma unroll
        for (int b = 0; b < BP; ++b) sum[b] += __builtin_nontemporal_load(src + b * R + r);
      }
      if (row < a.M) {
#pragma unroll
        for (int b = 0; b < BP; ++b)
          if (b < a.B) store_y(a, b, row, sum[b]);
      }
    }
    if (t == 0) __hip_atomic_store(a.counters + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// =====================================================================================================================
// Batch-1, mu = 8 kernel.
//
// One unit = (tile, super-chunk sc) = 256 virtual columns = chunks 2sc and 2sc+1, i.e. 32 sub-vectors of 8 columns.
// LDS table layout (floats): entry (p, buf, slot, s) at p*64 + buf*32 + slot*16 + s, where slot selects the chunk of
// the super-chunk and s the sub-vector of the chunk. A lane of row i reads its 16-byte entries with the byte rotation
// of the packed format: at step q it holds sub-vector (q + i) mod 16, and rows with (i mod 32) >= 16 see the two
// chunks swapped. So at every step the 32 lanes of a half-wavefront read 32 different (slot, s) columns of the table,
// i.e. 32 different LDS banks, whatever the patterns are.
// The byte address of a lookup, (p << 8) | (slot << 6) | (s << 2), is formed by one v_perm_b32 from the sign word and
// a per-lane constant; the buffer is an immediate offset.
// =====================================================================================================================

constexpr int kXvUnits = 12;  // units whose folded activations are staged in LDS at a time (1 KB each)

template <int NT, int RPT>
struct B1 {
  static constexpr int R = NT * RPT;
  static constexpr int NHI = NT / 32;                                   // p-ranges per (slot, s) in the build
  static constexpr int LO = NHI == 8 ? 5 : (NHI == 16 ? 4 : (NHI == 4 ? 6 : 7));
  static constexpr int E = 1 << LO;                                     // entries per thread per build
};

// Stage the folded activations xv = x[xidx] * colscale of the n units starting at super-chunk sc0 into
// xs[k*256 + col] (super-chunks wrap around at the end of a tile).
template <int NT>
__device__ __forceinline__ void stage_xv_b1(const GemmArgs& a, float* xs, int sc0, int n) {
  const int t = threadIdx.x;
  int sc = sc0;
  for (int k = 0; k < n; ++k) {
    for (int col = t; col < 256; col += NT) {
      const int v = sc * 256 + col;
      const uint16_t xi = a.xidx[v];
      const uint16_t cs = a.colscale[v];
      float val = 0.f;
      if (xi != 0xFFFFu) val = h2f(a.x[xi]) * h2f(cs);
      xs[k * 256 + col] = val;
    }
    if (++sc == a.steps) sc = 0;
  }
}

// Build the 2 x 16 tables (256 entries each) of one super-chunk into buffer BUF, from 256 staged activations.
// Thread t owns (slot, s) = ((t >> 4) & 1, t & 15) and the E patterns whose top bits equal t >> 5, enumerated in Gray
// order so that each entry is the previous one plus or minus 2*xv[n].
template <int NT, int BUF>
__device__ __forceinline__ void build_b1(float* lut, const float* xv256) {
  using P = B1<NT, 1>;
  const int t = threadIdx.x;
  const int slot = (t >> 4) & 1;
  const int s = t & 15;
  const int hi = t >> 5;
  const float4 lo4 = *reinterpret_cast<const float4*>(xv256 + slot * 128 + s * 8);
  const float4 hi4 = *reinterpret_cast<const float4*>(xv256 + slot * 128 + s * 8 + 4);
  const float xv[8] = {lo4.x, lo4.y, lo4.z, lo4.w, hi4.x, hi4.y, hi4.z, hi4.w};
  float v = 0.f;
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const bool plus = n >= P::LO && ((hi >> (n - P::LO)) & 1);
    v += plus ? xv[n] : -xv[n];
  }
  float d[8];
#pragma unroll
  for (int n = 0; n < 8; ++n) d[n] = 2.f * xv[n];
  float* col = lut + BUF * 32 + slot * 16 + s;
  const int pbase = hi << P::LO;
  col[pbase * 64] = v;
#pragma unroll
  for (int k = 1; k < P::E; ++k) {
    const int n = __builtin_ctz(k);
    const int g = k ^ (k >> 1);
    v += ((g >> n) & 1) ? d[n] : -d[n];
    col[(pbase | g) * 64] = v;
  }
}

template <int NT, int RPT>
__device__ __forceinline__ void load_unit_b1(const GemmArgs& a, int tile, int sc, uint32_t (&w)[RPT][8],
                                             float (&rs)[RPT][2], uint32_t hb) {
  using P = B1<NT, RPT>;
  const int t = threadIdx.x;
  const int32_t pa = a.chunk_plane[2 * sc];
  const int32_t pb = a.chunk_plane[2 * sc + 1];
  const int32_t p1 = hb ? pb : pa;
  const int32_t p2 = hb ? pa : pb;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int row = tile * P::R + t + NT * j;
    const int wave_row = tile * P::R + (t & ~63) + NT * j;
    if (wave_row < a.Mp) {
      const uint8_t* e0 = a.signs + (int64_t(2 * sc) * a.Mp + row) * 16;
      const uint8_t* e1 = a.signs + (int64_t(2 * sc + 1) * a.Mp + row) * 16;
      const uint4 v0 = load_stream16(e0);
      const uint4 v1 = load_stream16(e1);
      w[j][0] = v0.x; w[j][1] = v0.y; w[j][2] = v0.z; w[j][3] = v0.w;
      w[j][4] = v1.x; w[j][5] = v1.y; w[j][6] = v1.z; w[j][7] = v1.w;
      rs[j][0] = h2f(a.rscale[int64_t(p1) * a.Mp + row]);
      rs[j][1] = h2f(a.rscale[int64_t(p2) * a.Mp + row]);
    } else {
#pragma unroll
      for (int m = 0; m < 8; ++m) w[j][m] = 0u;
      rs[j][0] = 0.f;
      rs[j][1] = 0.f;
    }
  }
}

template <int BUF>
__device__ __forceinline__ float lds_at(const float* lut, uint32_t byte_addr) {
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(lut) + byte_addr + BUF * 128);
}

template <int NT, int RPT, int BUF>
__device__ __forceinline__ void lookup_b1(const float* lut, const uint32_t (&w)[RPT][8], const float (&rs)[RPT][2],
                                          const uint32_t (&c1)[4], const uint32_t (&c2)[4], float (&acc)[RPT][1]) {
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
        s1 += lds_at<BUF>(lut, __builtin_amdgcn_perm(w[j][m], c1[m], sel));
      }
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
        s2 += lds_at<BUF>(lut, __builtin_amdgcn_perm(w[j][4 + m], c2[m], sel));
      }
    }
    acc[j][0] = __builtin_fmaf(s1, rs[j][0], acc[j][0]);
    acc[j][0] = __builtin_fmaf(s2, rs[j][1], acc[j][0]);
  }
}

template <int NT, int RPT>
__global__ void __launch_bounds__(NT) k_gemv_mu8_b1(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) float lut[256 * 64];       // 64 KB, two buffers interleaved per pattern
  __shared__ __attribute__((aligned(16))) float xs[kXvUnits * 256];  // staged folded activations
  __shared__ int s_flag;

  const int t = threadIdx.x;
  const int64_t u0 = int64_t(blockIdx.x) * a.units / a.blocks;
  const int64_t u1 = (int64_t(blockIdx.x) + 1) * a.units / a.blocks;
  const int64_t first_tile = u0 / a.steps;

  // Per-lane byte offsets of the table columns read at step q: rows are congruent to t modulo 32.
  const uint32_t hb = (t >> 4) & 1u;
  uint32_t c1[4], c2[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    c1[m] = 0u;
    c2[m] = 0u;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const uint32_t s = (uint32_t(4 * m + bb) + uint32_t(t)) & 15u;
      c1[m] |= ((hb << 6) | (s << 2)) << (8 * bb);
      c2[m] |= (((hb ^ 1u) << 6) | (s << 2)) << (8 * bb);
    }
  }

  float acc[RPT][1];
#pragma unroll
  for (int j = 0; j < RPT; ++j) acc[j][0] = 0.f;
  uint32_t wA[RPT][8], wB[RPT][8];
  float rA[RPT][2], rB[RPT][2];

  // (tile, sc) of the current unit and of the next one, advanced without divisions
  const int steps = a.steps;
  int n_left = int(u1 - u0);           // units still to process, current one included
  int tile = int(first_tile);
  int sc = int(u0 - first_tile * steps);
  int tile_n = tile, sc_n = sc;
  auto advance = [&](int& tl, int& s) {
    if (++s == steps) { s = 0; ++tl; }
  };

  load_unit_b1<NT, RPT>(a, tile, sc, wA, rA, hb);
  int staged_left = n_left < kXvUnits ? n_left : kXvUnits;   // staged units not yet built, current one included
  int xs_pos = 0;                                             // slot of the current unit in xs
  stage_xv_b1<NT>(a, xs, sc, staged_left);
  __syncthreads();
  build_b1<NT, 0>(lut, xs);
  __syncthreads();

  while (true) {
    // ---- even step: current unit in buffer 0 / registers A ----
    tile_n = tile; sc_n = sc;
    advance(tile_n, sc_n);
    if (n_left > 1) {
      load_unit_b1<NT, RPT>(a, tile_n, sc_n, wB, rB, hb);
      if (--staged_left == 0) {
        staged_left = (n_left - 1) < kXvUnits ? (n_left - 1) : kXvUnits;
        stage_xv_b1<NT>(a, xs, sc_n, staged_left);
        xs_pos = -1;
        __syncthreads();
      }
      build_b1<NT, 1>(lut, xs + (xs_pos + 1) * 256);
    }
    lookup_b1<NT, RPT, 0>(lut, wA, rA, c1, c2, acc);
    if (sc == steps - 1 || n_left == 1) {
      finish_tile<NT, RPT, 1>(a, tile, first_tile, acc, &s_flag);
#pragma unroll
      for (int j = 0; j < RPT; ++j) acc[j][0] = 0.f;
    }
    __syncthreads();
    if (--n_left == 0) break;
    tile = tile_n; sc = sc_n; ++xs_pos;
    // ---- odd step: current unit in buffer 1 / registers B ----
    tile_n = tile; sc_n = sc;
    advance(tile_n, sc_n);
    if (n_left > 1) {
      load_unit_b1<NT, RPT>(a, tile_n, sc_n, wA, rA, hb);
      if (--staged_left == 0) {
        staged_left = (n_left - 1) < kXvUnits ? (n_left - 1) : kXvUnits;
        stage_xv_b1<NT>(a, xs, sc_n, staged_left);
        xs_pos = -1;
        __syncthreads();
      }
      build_b1<NT, 0>(lut, xs + (xs_pos + 1) * 256);
    }
    lookup_b1<NT, RPT, 1>(lut, wB, rB, c1, c2, acc);
    if (sc == steps - 1 || n_left == 1) {
      finish_tile<NT, RPT, 1>(a, tile, first_tile, acc, &s_flag);
#pragma unroll
      for (int j = 0; j < RPT; ++j) acc[j][0] = 0.f;
    }
    __syncthreads();
    if (--n_left == 0) break;
    tile = tile_n; sc = sc_n; ++xs_pos;
  }
}

// =====================================================================================================================
// Generic kernel: mu in {4, 8}, any batch (1..16).
//
// One unit = (tile, chunk c, batch group g): 128 virtual columns, BG batch rows. LDS table layout (floats): entry
// (p, s, b) at ((p * SPC + s) * BG + b) within a buffer, SPC = 128/mu sub-vectors per chunk, so the BG batch values of
// one lookup are contiguous (one ds_read of 4*BG bytes). A lane of row i reads sub-vector (q + i) mod SPC at step q.
// Each sign word is loaded once per chunk and reused for every batch group of that chunk.
// =====================================================================================================================

template <int MU, int BG, int NG, int NT, int RPT>
struct Gen {
  static constexpr int SPC = 128 / MU;          // sub-vectors per chunk
  static constexpr int NP = 1 << MU;            // patterns
  static constexpr int BP = BG * NG;            // padded batch
  static constexpr int R = NT * RPT;
  static constexpr int TBL = NP * SPC * BG;     // floats per table buffer
  static constexpr int XV = 128 * BG;           // staged activations per unit
  static constexpr int XU = 8;                  // units staged at a time
  static constexpr int GROUPS = NT / SPC;       // pattern ranges in the build
  static constexpr int PER = NP / GROUPS;       // patterns per thread in the build (a power of two)
  static constexpr int LOB = PER == 16 ? 4 : (PER == 8 ? 3 : (PER == 4 ? 2 : (PER == 2 ? 1 : 0)));
};

template <int BG>
__device__ __forceinline__ void read_vec(const float* p, float (&f)[BG]);
template <>
__device__ __forceinline__ void read_vec<1>(const float* p, float (&f)[1]) { f[0] = *p; }
template <>
__device__ __forceinline__ void read_vec<2>(const float* p, float (&f)[2]) {
  const float2 v = *reinterpret_cast<const float2*>(p);
  f[0] = v.x; f[1] = v.y;
}
template <>
__device__ __forceinline__ void read_vec<4>(const float* p, float (&f)[4]) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
}

// Stage the folded activations of n units starting at (c, g) into xs[k*XV + col*BG + b].
template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void stage_xv_gen(const GemmArgs& a, float* xs, int c, int g, int n) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  const int t = threadIdx.x;
  for (int k = 0; k < n; ++k) {
    for (int e = t; e < P::XV; e += NT) {
      const int col = e / BG;
      const int b = e % BG;
      const int bat = g * BG + b;
      const int v = c * 128 + col;
      const uint16_t xi = a.xidx[v];
      float val = 0.f;
      if (xi != 0xFFFFu && bat < a.B) val = h2f(a.x[int64_t(bat) * a.ldx + xi]) * h2f(a.colscale[v]);
      xs[k * P::XV + e] = val;
    }
    if (++g == NG) {
      g = 0;
      if (++c == a.NCP) c = 0;
    }
  }
}

// Build the SPC tables of one chunk for BG batch rows. Thread t owns sub-vector s = t % SPC and the PER patterns whose
// high bits are t / SPC, enumerated in Gray order (each entry is the previous one plus or minus 2*xv[n]).
template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void build_gen(float* tbl, const float* xs) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  const int t = threadIdx.x;
  const int s = t % P::SPC;
  const int grp = t / P::SPC;
#pragma unroll
  for (int b = 0; b < BG; ++b) {
    float xv[MU];
#pragma unroll
    for (int n = 0; n < MU; ++n) xv[n] = xs[(s * MU + n) * BG + b];
    float v = 0.f;
#pragma unroll
    for (int n = 0; n < MU; ++n) {
      const bool plus = n >= P::LOB && ((grp >> (n - P::LOB)) & 1);
      v += plus ? xv[n] : -xv[n];
    }
    const int pbase = grp << P::LOB;
    tbl[(pbase * P::SPC + s) * BG + b] = v;
#pragma unroll
    for (int k = 1; k < P::PER; ++k) {
      const int n = __builtin_ctz(k);
      const int gk = k ^ (k >> 1);
      v += ((gk >> n) & 1) ? 2.f * xv[n] : -2.f * xv[n];
      tbl[((pbase | gk) * P::SPC + s) * BG + b] = v;
    }
  }
}

template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void load_unit_gen(const GemmArgs& a, int tile, int c, uint32_t (&w)[RPT][4],
                                              float (&rs)[RPT]) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  const int t = threadIdx.x;
  const int32_t plane = a.chunk_plane[c];
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int row = tile * P::R + t + NT * j;
    const int wave_row = tile * P::R + (t & ~63) + NT * j;
    if (wave_row < a.Mp) {
      const int h = (MU == 8) ? ((c & 1) ^ ((row & 31) >= 16 ? 1 : 0)) : (c & 1);
      const uint4 v = load_stream16(a.signs + ((int64_t(c >> 1) * 2 + h) * a.Mp + row) * 16);
      w[j][0] = v.x; w[j][1] = v.y; w[j][2] = v.z; w[j][3] = v.w;
      rs[j] = h2f(a.rscale[int64_t(plane) * a.Mp + row]);
    } else {
      w[j][0] = w[j][1] = w[j][2] = w[j][3] = 0u;
      rs[j] = 0.f;
    }
  }
}

template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void lookup_gen(const float* tbl, const uint32_t (&w)[RPT][4], const float (&rs)[RPT], int g,
                                           float (&acc)[RPT][BG * NG]) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  const uint32_t t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    float sum[BG];
#pragma unroll
    for (int b = 0; b < BG; ++b) sum[b] = 0.f;
#pragma unroll
    for (int q = 0; q < P::SPC; ++q) {
      const uint32_t p = (w[j][q / (32 / MU)] >> (MU * (q % (32 / MU)))) & uint32_t(P::NP - 1);
      const uint32_t sv = (uint32_t(q) + t) & uint32_t(P::SPC - 1);
      float f[BG];
      read_vec<BG>(tbl + (p * P::SPC + sv) * BG, f);
#pragma unroll
      for (int b = 0; b < BG; ++b) sum[b] += f[b];
    }
#pragma unroll
    for (int gg = 0; gg < NG; ++gg) {
#pragma unroll
      for (int b = 0; b < BG; ++b) {
        const float upd = __builtin_fmaf(sum[b], rs[j], acc[j][gg * BG + b]);
        acc[j][gg * BG + b] = (gg == g) ? upd : acc[j][gg * BG + b];
      }
    }
  }
}

template <int MU, int BG, int NG, int NT, int RPT>
__global__ void __launch_bounds__(NT) k_gemm_generic(GemmArgs a) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  __shared__ __attribute__((aligned(16))) float tbl[2 * P::TBL];
  __shared__ __attribute__((aligned(16))) float xs[P::XU * P::XV];
  __shared__ int s_flag;

  const int64_t u0 = int64_t(blockIdx.x) * a.units / a.blocks;
  const int64_t u1 = (int64_t(blockIdx.x) + 1) * a.units / a.blocks;
  const int64_t first_tile = u0 / a.steps;
  const int rem0 = int(u0 - first_tile * a.steps);

  float acc[RPT][P::BP];
#pragma unroll
  for (int j = 0; j < RPT; ++j)
#pragma unroll
    for (int b = 0; b < P::BP; ++b) acc[j][b] = 0.f;
  uint32_t w[RPT][4], wn[RPT][4];
  float rs[RPT], rsn[RPT];

  int n_left = int(u1 - u0);
  int tile = int(first_tile), c = rem0 / NG, g = rem0 % NG;
  load_unit_gen<MU, BG, NG, NT, RPT>(a, tile, c, w, rs);
  int staged_left = n_left < P::XU ? n_left : P::XU;
  int xs_pos = 0;
  stage_xv_gen<MU, BG, NG, NT, RPT>(a, xs, c, g, staged_left);
  __syncthreads();
  build_gen<MU, BG, NG, NT, RPT>(tbl, xs);
  __syncthreads();

  int buf = 0;
  while (true) {
    int tile_n = tile, c_n = c, g_n = g + 1;
    if (g_n == NG) {
      g_n = 0;
      if (++c_n == a.NCP) { c_n = 0; ++tile_n; }
    }
    const bool has_next = n_left > 1;
    const bool new_chunk = has_next && g_n == 0;
    if (has_next) {
      if (--staged_left == 0) {
        staged_left = (n_left - 1) < P::XU ? (n_left - 1) : P::XU;
        stage_xv_gen<MU, BG, NG, NT, RPT>(a, xs, c_n, g_n, staged_left);
        xs_pos = -1;
        __syncthreads();
      }
      build_gen<MU, BG, NG, NT, RPT>(tbl + (buf ^ 1) * P::TBL, xs + (xs_pos + 1) * P::XV);
      if (new_chunk) load_unit_gen<MU, BG, NG, NT, RPT>(a, tile_n, c_n, wn, rsn);
    }
    lookup_gen<MU, BG, NG, NT, RPT>(tbl + buf * P::TBL, w, rs, g, acc);
    if ((c == a.NCP - 1 && g == NG - 1) || n_left == 1) {
      finish_tile<NT, RPT, P::BP>(a, tile, first_tile, acc, &s_flag);
#pragma unroll
      for (int j = 0; j < RPT; ++j)
#pragma unroll
        for (int b = 0; b < P::BP; ++b) acc[j][b] = 0.f;
    }
    __syncthreads();
    if (--n_left == 0) break;
    if (new_chunk) {
#pragma unroll
      for (int j = 0; j < RPT; ++j) {
        w[j][0] = wn[j][0]; w[j][1] = wn[j][1]; w[j][2] = wn[j][2]; w[j][3] = wn[j][3];
        rs[j] = rsn[j];
      }
    }
    tile = tile_n; c = c_n; g = g_n; ++xs_pos;
    buf ^= 1;
  }
}

// =====================================================================================================================
// Launch
// =====================================================================================================================

template <int NT, int RPT>
static void launch_b1(const GemmArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((k_gemv_mu8_b1<NT, RPT>), dim3(unsigned(a.blocks)), dim3(NT), 0, stream, a);
}

template <int MU, int BG, int NG>
static bool launch_gen_rpt(const GemmArgs& a, int rpt, hipStream_t stream) {
  switch (rpt) {
    case 1: hipLaunchKernelGGL((k_gemm_generic<MU, BG, NG, 256, 1>), dim3(unsigned(a.blocks)), dim3(256), 0, stream, a); return true;
    case 2: hipLaunchKernelGGL((k_gemm_generic<MU, BG, NG, 256, 2>), dim3(unsigned(a.blocks)), dim3(256), 0, stream, a); return true;
    case 4:
      if constexpr (BG * NG <= 2 && MU == 8) {
        hipLaunchKernelGGL((k_gemm_generic<MU, BG, NG, 256, 4>), dim3(unsigned(a.blocks)), dim3(256), 0, stream, a);
        return true;
      }
      return false;
  }
  return false;
}

template <int MU>
static bool launch_gen_mu(const GemmArgs& a, const Plan& p, hipStream_t stream) {
  if (p.bg == 1 && p.n_groups == 1) return launch_gen_rpt<MU, 1, 1>(a, p.rpt, stream);
  if (p.bg == 2 && p.n_groups == 1) return launch_gen_rpt<MU, 2, 1>(a, p.rpt, stream);
  if (p.bg == 4 && p.n_groups == 1) return launch_gen_rpt<MU, 4, 1>(a, p.rpt, stream);
  if (p.bg == 4 && p.n_groups == 2) return launch_gen_rpt<MU, 4, 2>(a, p.rpt, stream);
  if (p.bg == 4 && p.n_groups == 4) return launch_gen_rpt<MU, 4, 4>(a, p.rpt, stream);
  return false;
}

fluxbin_status launch_gemm(const fluxbin_layer& L, const Plan& p, int B, const uint16_t* d_x, int64_t ldx, void* d_y,
                           int64_t ldy, int y_fp32, void* d_ws, hipStream_t stream) {
  GemmArgs a{};
  const uint8_t* base = static_cast<const uint8_t*>(L.d_base);
  a.signs = base + L.off_signs;
  a.rscale = reinterpret_cast<const uint16_t*>(base + L.off_rscale);
  a.colscale = reinterpret_cast<const uint16_t*>(base + L.off_colscale);
  a.xidx = reinterpret_cast<const uint16_t*>(base + L.off_xidx);
  a.chunk_plane = reinterpret_cast<const int32_t*>(base + L.off_chunk_plane);
  a.x = d_x;
  a.y = d_y;
  a.counters = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(d_ws) + p.ws_counters_off);
  a.partials = reinterpret_cast<float*>(static_cast<uint8_t*>(d_ws) + p.ws_partials_off);
  a.ldx = ldx;
  a.ldy = ldy;
  a.units = p.units;
  a.blocks = p.blocks;
  a.M = int32_t(L.shape.M);
  a.Mp = int32_t(L.Mp);
  a.NSC = int32_t(L.NSC);
  a.NCP = int32_t(2 * L.NSC);
  a.steps = int32_t(p.units / p.n_tiles);
  a.B = B;
  a.y_fp32 = y_fp32;
  a.n_tiles = int32_t(p.n_tiles);
  bool ok = true;
  if (p.kernel == 0) {
    switch (p.rpt) {
      case 1: launch_b1<256, 1>(a, stream); break;
      case 2: launch_b1<256, 2>(a, stream); break;
      case 4: launch_b1<256, 4>(a, stream); break;
      default: ok = false;
    }
  } else if (L.shape.mu == 8) {
    ok = launch_gen_mu<8>(a, p, stream);
  } else {
    ok = launch_gen_mu<4>(a, p, stream);
  }
  if (!ok) return fail(FLUXBIN_ERR_UNSUPPORTED, "no kernel instance for this launch plan");
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the LUT-GEMM kernel");
  return FLUXBIN_OK;
}

}  // namespace fluxbin
