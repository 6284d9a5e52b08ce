// Small-batch (B = 2..16) product of libfluxbin on the gfx950 matrix cores (MFMA).
//
// What is computed is the same as the LUT kernels (Eqs. 10-11 and 15), for every batch row b < B:
//   y[b, i] = sum_c rscale[plane(c)][i] * sum_{v in chunk c} s(i, v) * colscale[v] * x[b, xidx[v]],
// s(i, v) = +1 for a set sign bit and -1 for a clear one. The LUT kernels form the inner sum by table lookups, whose
// cost grows with the batch (one table entry read and added per batch row and sub-vector). With B > 1 the same inner
// sums are a dense contraction over the virtual columns: a (rows x 128) block of signed column scales times a
// (128 x B) block of activations. Here every 32 columns of that contraction are one v_mfma_f32_16x16x32_f16, and the
// cost per sign bit is the same for any B <= 16 (the batch occupies the 16 columns of the MFMA tile).
//
// Exactness. The A operand is s(i, v) * |colscale[v]|, an fp16 value (the column scale with its sign bit replaced),
// and the B operand is x[b, xidx[v]] with the sign of colscale[v] folded in, also fp16. Their products are exact in
// the fp32 accumulation of the matrix core, as x * colscale is exact in fp32 for the LUT kernels (two 11-bit
// significands). The row scale multiplies each 128-column chunk's fp32 sum once (Eq. 15's order), and y is the fp32
// sum over chunks. Padding columns have column scale 0 and stage x = 0, so they add exactly zero.
//
// Sign decode. By the packed format, row i's 16-byte entry of a chunk holds the chunk's 128 sign bits rotated left by
// R(i) bits (mu = 8: R = 8 (i mod 16); mu = 4: R = 4 (i mod 32)). Lane (r, g) of a 16-row MFMA block needs canonical
// bits 32g .. 32g+31 of its row r: two 32-bit words of the entry and one funnel shift give them, whatever the
// rotation. The K dimension of the contraction is ordered so that element pair k of K step q holds canonical columns
// (32g + 4q + k, 32g + 4q + k + 16): a left shift of the 32 bits by 15 - (4q + k) puts both sign bits at bit
// positions 15 and 31, the fp16 sign bits of the pair, so one and-or with the column-scale pair forms the operand
// (a set bit gives -|colscale|, so the matrix core sums -s; the row scale is applied negated). The words of two row
// blocks are shifted together as one 64-bit value.
//
// Work decomposition (as in the LUT kernels): a tile is 256 rows, 64 per wavefront of a 256-thread workgroup (four
// 16-row MFMA blocks); a unit is a tile times a super-chunk (256 virtual columns, both stored chunk slots); units are
// numbered tile-major, split into contiguous equal ranges, one per workgroup; split tiles are reduced by the
// deterministic counter protocol of fluxbin_device.h (same partial-sum layout, so its reduction code is shared).
//
// Memory pipeline. Each lane requests its row's whole 16-byte entries of a unit (one 16-byte load per chunk) and one
// 32-bit word of row scales, D units ahead of the unit being multiplied (2 KB of signs per wavefront per unit, no
// byte requested twice); a wavefront passes the entries to its MFMA lanes through its own LDS scratch. The
// activations of a unit (gathered through the VCM index table) are requested together with its signs, because
// vector loads complete in issue order: a load issued after the sign loads of a later unit could only be used once
// those had arrived. They are written to a double-buffered LDS staging area one unit before they are multiplied.
#include <hip/hip_runtime.h>

#include "fluxbin_device.h"

namespace fluxbin {

namespace {

typedef _Float16 mf_half8 __attribute__((ext_vector_type(8)));
typedef float mf_float4 __attribute__((ext_vector_type(4)));
typedef unsigned int mf_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int mf_u32x2 __attribute__((ext_vector_type(2)));

constexpr int kMfNT = 256;                          // threads per workgroup: four wavefronts of 64 rows
constexpr int kMfR = 256;                           // rows per tile
constexpr int kMfXStride = 68;                      // dwords per (chunk, column group, K step) block: 64 + 4 pad
constexpr int kMfXUnit = 2 * 4 * 4 * kMfXStride;    // dwords of staged activation pairs per unit
constexpr int kMfAUnit = 2 * 4 * 16;                // dwords of column-scale pairs per unit
constexpr int kMfScr = 64 * 8;                      // dwords of a wavefront's sign scratch: 64 rows x 32 bytes
constexpr int kMfTStride = 68;                      // dwords per batch row of a wavefront's tile-end transpose
constexpr int kMfScrWave = 16 * kMfTStride;         // dwords of a wavefront's scratch (>= kMfScr + 64 row scales)
static_assert(kMfScrWave >= kMfScr + 64, "scratch too small");

// Requested data of one unit: the lane's row entries of both chunks (lane l: row 16 (l >> 4) + (l & 15) of the
// wavefront's 64 rows), one word of row scales (lane l: rows 2 (l & 31) and 2 (l & 31) + 1 of chunk l >> 5), and the
// lane's staged column: its metadata and x of batch rows 0..BP-1.
template <int BP>
struct MfUnitRegs {
  mf_u32x4 e[2];
  uint32_t r;
  uint32_t meta;        // xidx | colscale << 16 (thread t owns virtual column t of the unit)
  uint32_t xv[BP];      // x bits of batch rows 0..BP-1, one register each (rows >= B read row B-1)
};

struct MfCursor {
  int tile, sc;
};

__device__ __forceinline__ void mf_advance(const GemmArgs& a, MfCursor& c) {
  if (++c.sc == a.steps) {
    c.sc = 0;
    ++c.tile;
  }
}

// First row of 16-row block rb of wavefront `wave` in `tile`, moved back inside the padded rows when the tile extends
// past them (such rows are never stored: their y rows are >= M).
__device__ __forceinline__ uint32_t mf_block_row(const GemmArgs& a, int tile, int wave, int rb) {
  const int r = tile * kMfR + wave * 64 + 16 * rb;
  return uint32_t(r <= a.Mp - 16 ? r : a.Mp - 16);
}

__device__ __forceinline__ uint32_t mf_load_meta(const GemmArgs& a, int sc, int t) {
  const int v = sc * 256 + t;
  return uint32_t(a.xidx[v]) | (uint32_t(a.colscale[v]) << 16);
}

// Requests unit c's data into u: activations first (u.meta must hold the unit's metadata), then the sign entries and
// row scales. p0, p1: row-scale planes of the unit's two chunks.
template <int BP, int MU>
__device__ __forceinline__ void mf_issue(const GemmArgs& a, const MfCursor& c, int32_t p0, int32_t p1, int wave,
                                         int lane, const uint16_t* const (&xrow)[BP], MfUnitRegs<BP>& u) {
  {
    const uint32_t xi = u.meta & 0xFFFFu;
    const uint32_t col = xi == 0xFFFFu ? 0u : xi;
#pragma unroll
    for (int b = 0; b < BP; ++b) u.xv[b] = xrow[b][col];
  }
  const int rbl = lane >> 4;
  const uint32_t row = mf_block_row(a, c.tile, wave, rbl) + uint32_t(lane & 15);
  const int64_t plane_bytes = int64_t(a.Mp) * 16;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    // mu = 8 stores the two chunks of a super-chunk swapped for rows with i mod 32 >= 16, i.e. odd row blocks
    const int slot = MU == 8 ? (h ^ (rbl & 1)) : h;
    u.e[h] = __builtin_nontemporal_load(
        reinterpret_cast<const mf_u32x4*>(a.signs + int64_t(2 * c.sc) * plane_bytes + (slot ? plane_bytes : 0) +
                                          row * 16u));
  }
  const int p = lane & 31;   // rows 2p, 2p + 1 of the wavefront: block p >> 3, rows (2p) & 15 and the next
  const uint32_t rrow = mf_block_row(a, c.tile, wave, p >> 3) + uint32_t((2 * p) & 15);
  const int32_t plane = lane < 32 ? p0 : p1;
  u.r = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint8_t*>(a.rscale) +
                                           (int64_t(plane) * a.Mp + rrow) * 2);
}

// Writes a staged unit: the activation pairs (sign of the column scale folded in; 0 for padding columns, so that x is
// never multiplied there, not even by a zero) and the column-scale pairs (magnitudes) in the order the MFMA operands
// read them. Batch rows b >= B hold row B-1's values: MFMA output column b depends on activation column b only, and
// columns >= B are never stored.
template <int BP>
__device__ __forceinline__ void mf_stage_write(const GemmArgs& a, const MfUnitRegs<BP>& u, uint32_t* sx, uint32_t* sa,
                                               int t) {
  const int h = t >> 7, cc = t & 127, g = cc >> 5, m = cc & 31, j = m & 15, hf = m >> 4;
  const int q = j >> 2, k = j & 3;
  const uint32_t xi = u.meta & 0xFFFFu;
  const uint16_t cs = uint16_t(u.meta >> 16);
  const uint16_t flip = cs & 0x8000u;
  const uint16_t keep = xi != 0xFFFFu ? uint16_t(0xFFFFu) : uint16_t(0);
  uint16_t* sx16 = reinterpret_cast<uint16_t*>(sx);
  const int base = ((h * 4 + g) * 4 + q) * kMfXStride + k;
#pragma unroll
  for (int b = 0; b < BP; ++b) sx16[(base + 4 * b) * 2 + hf] = uint16_t((uint16_t(u.xv[b]) ^ flip) & keep);
  reinterpret_cast<uint16_t*>(sa)[((h * 4 + g) * 16 + j) * 2 + hf] = uint16_t(cs & 0x7FFFu);
}

// 64-bit left shift by a constant, as one v_lshlrev_b64: it shifts two 32-bit words in the time a 32-bit shift takes
// one (measured on gfx950). Written as an instruction because the compiler, seeing that only bits 15 and 31 of each
// half are used, would split it back into two 32-bit shifts. For {w_hi : w_lo} << s (s <= 15), bits 15 and 31 of each
// half are bits 15 - s and 31 - s of its own word: the bits the low word pushes into the high half land below bit 15.
__device__ __forceinline__ uint64_t mf_shl64(uint64_t v, uint32_t s) {
  uint64_t r;
  asm("v_lshlrev_b64 %0, %1, %2" : "=v"(r) : "s"(s), "v"(v));
  return r;
}

// Multiplies one staged unit into the accumulators. xs/as: the unit's staged activation and column-scale pairs;
// scr: the wavefront's sign scratch (32 bytes per row: the 16-byte entry, then its first 8 bytes again, so that the two
// words a lane reads never wrap), followed by 64 words of row scales.
template <bool SHL64>
__device__ __forceinline__ void mf_unit(const uint32_t* xs, const uint32_t* as, const mf_u32x4 (&e)[2], uint32_t r,
                                        uint32_t* scr, int lane, int r16, int g, const uint32_t (&aw)[2], uint32_t sh,
                                        float (&acc)[4][4]) {
  uint32_t* srs = scr + kMfScr;
  srs[lane] = r;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    *reinterpret_cast<mf_u32x4*>(scr + lane * 8) = e[h];
    *reinterpret_cast<mf_u32x2*>(scr + lane * 8 + 4) = mf_u32x2{e[h][0], e[h][1]};
    uint32_t w[4];
    uint2 rs[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const uint32_t* ent = scr + (16 * rb + r16) * 8 + aw[rb & 1];
      w[rb] = __builtin_amdgcn_alignbit(ent[1], ent[0], sh);
      rs[rb] = *reinterpret_cast<const uint2*>(srs + h * 32 + 8 * rb + 2 * g);
    }
    // the words of row blocks 2rp and 2rp + 1 as one 64-bit value (high: 2rp + 1), shifted together below
    uint64_t w2[2] = {0, 0};
    if constexpr (SHL64) {
      w2[0] = (uint64_t(w[1]) << 32) | w[0];
      w2[1] = (uint64_t(w[3]) << 32) | w[2];
    }
    mf_float4 tmp[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const mf_u32x4 bx = *reinterpret_cast<const mf_u32x4*>(xs + ((h * 4 + g) * 4 + q) * kMfXStride + 4 * r16);
      const mf_u32x4 ac = *reinterpret_cast<const mf_u32x4*>(as + (h * 4 + g) * 16 + 4 * q);
#pragma unroll
      for (int rp = 0; rp < 2; ++rp) {
        mf_u32x4 av0, av1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t s = uint32_t(15 - (4 * q + k));
          if constexpr (SHL64) {
            const uint64_t sft = mf_shl64(w2[rp], s);
            av0[k] = (uint32_t(sft) & 0x80008000u) | ac[k];
            av1[k] = (uint32_t(sft >> 32) & 0x80008000u) | ac[k];
          } else {
            av0[k] = ((w[2 * rp] << s) & 0x80008000u) | ac[k];
            av1[k] = ((w[2 * rp + 1] << s) & 0x80008000u) | ac[k];
          }
        }
        const mf_float4 c0 = q == 0 ? mf_float4{0.f, 0.f, 0.f, 0.f} : tmp[2 * rp];
        const mf_float4 c1 = q == 0 ? mf_float4{0.f, 0.f, 0.f, 0.f} : tmp[2 * rp + 1];
        tmp[2 * rp] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mf_half8, av0),
                                                             __builtin_bit_cast(mf_half8, bx), c0, 0, 0, 0);
        tmp[2 * rp + 1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mf_half8, av1),
                                                                 __builtin_bit_cast(mf_half8, bx), c1, 0, 0, 0);
      }
    }
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      acc[rb][0] = fmaf(-h2f(uint16_t(rs[rb].x)), tmp[rb][0], acc[rb][0]);
      acc[rb][1] = fmaf(-h2f(uint16_t(rs[rb].x >> 16)), tmp[rb][1], acc[rb][1]);
      acc[rb][2] = fmaf(-h2f(uint16_t(rs[rb].y)), tmp[rb][2], acc[rb][2]);
      acc[rb][3] = fmaf(-h2f(uint16_t(rs[rb].y >> 16)), tmp[rb][3], acc[rb][3]);
    }
  }
}

// End of a tile's contribution: y for a tile only this workgroup covers, else its partial sums (slot 0 for the
// workgroup's first tile, 1 for its last), in the layout reduce_tile reads: element (b, row in tile) at b * R + row.
// Lane (b = r16, g) holds rows 16 rb + 4 g + v of the wavefront's 64; the wavefront first transposes them through its
// LDS scratch (row block rb of batch row b at b * kMfTStride + 16 rb), so that every store instruction writes 64
// consecutive rows of one batch row (whole memory lines: scattered 4-byte stores wrote each line several times).
template <int BP>
__device__ __forceinline__ void mf_tile_end(const GemmArgs& a, int tile, bool shared, int slot, int wave, int lane,
                                            int r16, int g, const float (&acc)[4][4], uint32_t* scr) {
  float* t = reinterpret_cast<float*>(scr);
  if (r16 < BP) {
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
      *reinterpret_cast<mf_float4*>(t + r16 * kMfTStride + 16 * rb + 4 * g) =
          mf_float4{acc[rb][0], acc[rb][1], acc[rb][2], acc[rb][3]};
  }
  if (shared) {
    float* mine = a.partials + ((int64_t(blockIdx.x) * 2 + slot) * BP) * kMfR + wave * 64 + lane;
#pragma unroll
    for (int b = 0; b < BP; ++b)
      __hip_atomic_store(mine + b * kMfR, t[b * kMfTStride + lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    const int64_t row = int64_t(tile) * kMfR + wave * 64 + lane;
    if (row < a.M) {
#pragma unroll
      for (int b = 0; b < BP; ++b)
        if (b < a.B) store_y(a, b, row, t[b * kMfTStride + lane]);
    }
  }
}

template <int BP, int MU, int D>
struct MfKernel {
  struct State {
    int n;
    int first_tile, last_tile;
    bool first_shared, last_shared;
    int n_pending;
    MfCursor cur;    // unit K
    MfCursor nxt;    // unit K + D (clamped to the last unit of the range)
    int stg_sc;      // super-chunk of unit K + D + 1 (clamped), whose metadata is requested next
    float acc[4][4];
  };

  struct Lane {
    int t, lane, wave, r16, g;
    uint32_t aw[2];   // word index, within a row's entry, of the first word holding the lane's canonical bits
    uint32_t sh;      // funnel shift
  };

  // Unit K of the workgroup (compile-time K < kMfMaxUnits; the launch plan keeps the range within that), with
  // register set K mod (D + 1). Fully unrolled, so no loads are carried through a loop header.
  // Order: request unit K+D (activations, then signs and row scales) and the metadata of unit K+D+1; multiply unit K
  // (waits only for its own data, requested D units ago); stage unit K+1 (requested D-1 units ago); end a tile.
  template <int K>
  __device__ static __forceinline__ void step(const GemmArgs& a, State& s, MfUnitRegs<BP> (&ur)[D + 1],
                                              uint32_t& meta_next, const int* s_planes, uint32_t* sx, uint32_t* sa,
                                              uint32_t* scr, const Lane& ln, const uint16_t* const (&xrow)[BP]) {
    if constexpr (K < kMfMaxUnits) {
      if (K >= s.n) return;
      constexpr int P = K % (D + 1);
      constexpr int PN = (K + D) % (D + 1);
      constexpr int PS = (K + 1) % (D + 1);
      {
        const int kd = K + D < s.n ? K + D : s.n - 1;
        ur[PN].meta = meta_next;
        mf_issue<BP, MU>(a, s.nxt, s_planes[2 * kd], s_planes[2 * kd + 1], ln.wave, ln.lane, xrow, ur[PN]);
        meta_next = mf_load_meta(a, s.stg_sc, ln.t);
        if (K + D + 1 < s.n) mf_advance(a, s.nxt);
        if (K + D + 2 < s.n && ++s.stg_sc == a.steps) s.stg_sc = 0;
      }
      __builtin_amdgcn_sched_barrier(0);
      // 64-bit shifts free VALU issue slots; with 16 batch rows their register pairs would spill
      mf_unit<(BP <= 8)>(sx + (K & 1) * kMfXUnit, sa + (K & 1) * kMfAUnit, ur[P].e, ur[P].r, scr, ln.lane, ln.r16, ln.g, ln.aw,
              ln.sh, s.acc);
      if (K + 1 < s.n)
        mf_stage_write<BP>(a, ur[PS], sx + ((K + 1) & 1) * kMfXUnit, sa + ((K + 1) & 1) * kMfAUnit, ln.t);
      if (s.cur.sc == a.steps - 1 || K + 1 == s.n) {
        const int tile = s.cur.tile;
        const bool shared = tile == s.first_tile ? s.first_shared : (tile == s.last_tile && s.last_shared);
        mf_tile_end<BP>(a, tile, shared, tile == s.first_tile ? 0 : 1, ln.wave, ln.lane, ln.r16, ln.g, s.acc, scr);
        if (shared) ++s.n_pending;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
          for (int v = 0; v < 4; ++v) s.acc[rb][v] = 0.f;
      }
      mf_advance(a, s.cur);
      __syncthreads();
      step<K + 1>(a, s, ur, meta_next, s_planes, sx, sa, scr, ln, xrow);
    }
  }
};

template <int BP, int MU, int D, bool R2>
__global__ void __launch_bounds__(kMfNT, 3) k_gemm_mfma(GemmArgs a) {
  using K = MfKernel<BP, MU, D>;
  __shared__ __attribute__((aligned(16))) uint32_t sx[2 * kMfXUnit];
  __shared__ __attribute__((aligned(16))) uint32_t sa[2 * kMfAUnit];
  __shared__ __attribute__((aligned(16))) uint32_t scr_all[4 * kMfScrWave];
  __shared__ int s_planes[2 * kMfMaxUnits];
  __shared__ int s_flag;

  typename K::Lane ln;
  ln.t = threadIdx.x;
  ln.lane = ln.t & 63;
  ln.wave = ln.t >> 6;
  ln.r16 = ln.lane & 15;
  ln.g = ln.lane >> 4;
  // Words of a row's entry that hold canonical bits 32g..32g+31: they start at stored bit (32g - R) mod 128;
  // mu = 4: index 1 for odd row blocks (rows with i mod 32 >= 16 rotate by 64 more bits).
  {
    const int rot0 = MU == 8 ? 8 * ln.r16 : 4 * ln.r16;
#pragma unroll
    for (int par = 0; par < 2; ++par)
      ln.aw[par] = uint32_t(((32 * ln.g - rot0 - (MU == 4 ? 64 * par : 0)) & 127) >> 5);
    ln.sh = uint32_t((32 * ln.g - rot0) & 31);
  }
  uint32_t* scr = scr_all + ln.wave * kMfScrWave;

  const int u0 = first_unit(a, blockIdx.x);
  const int u1 = first_unit(a, blockIdx.x + 1);
  typename K::State s;
  s.n = u1 - u0;
  s.cur.tile = u0 / a.steps;
  s.cur.sc = u0 - s.cur.tile * a.steps;
  s.first_tile = s.cur.tile;
  s.last_tile = (u1 - 1) / a.steps;
  s.first_shared = tile_is_shared(a, s.first_tile);
  s.last_shared = tile_is_shared(a, s.last_tile);
  s.n_pending = 0;
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int v = 0; v < 4; ++v) s.acc[rb][v] = 0.f;

  // Row-scale planes of the range's chunks (the launch plan keeps n <= kMfMaxUnits), and metadata of units 0..D.
  if (ln.t < 2 * s.n) {
    int sc = s.cur.sc + (ln.t >> 1);
    while (sc >= a.steps) sc -= a.steps;
    s_planes[ln.t] = a.chunk_plane[2 * sc + (ln.t & 1)];
  }
  // Batch rows of x (wave-uniform; rows >= B read row B-1, masked when staged).
  const uint16_t* xrow[BP];
#pragma unroll
  for (int b = 0; b < BP; ++b) xrow[b] = a.x + int64_t(b < a.B ? b : a.B - 1) * a.ldx;
  MfUnitRegs<BP> ur[D + 1];
  uint32_t meta_next;
  {
    int sc = s.cur.sc;
#pragma unroll
    for (int k = 0; k <= D; ++k) {
      const uint32_t m = mf_load_meta(a, sc, ln.t);
      if (k < D)
        ur[k].meta = m;
      else
        meta_next = m;
      if (k + 1 < s.n && ++sc == a.steps) sc = 0;
    }
    s.stg_sc = sc;   // unit D + 1 (clamped)
  }
  // Staged rows of batch rows >= BP stay zero for the whole launch.
  for (int i = ln.t; i < 2 * kMfXUnit; i += kMfNT) sx[i] = 0u;
  __syncthreads();   // planes in LDS; zero fill done before any staged value is written
  s.nxt = s.cur;
#pragma unroll
  for (int k = 0; k < D; ++k) {
    const int kk = k < s.n ? k : s.n - 1;
    mf_issue<BP, MU>(a, s.nxt, s_planes[2 * kk], s_planes[2 * kk + 1], ln.wave, ln.lane, xrow, ur[k]);
    if (k + 1 < s.n) mf_advance(a, s.nxt);
  }
  mf_stage_write<BP>(a, ur[0], sx, sa, ln.t);
  __syncthreads();
  K::template step<0>(a, s, ur, meta_next, s_planes, sx, sa, scr, ln, xrow);
  if constexpr (!R2) {
    const int pend0 = s.first_shared ? s.first_tile : s.last_tile;
    publish_pending<kMfNT, 1, BP>(a, pend0, s.last_tile, s.n_pending, &s_flag);
  }
}

template <int BP, int D, bool R2>
bool launch_mfma_bp(const GemmArgs& a, int mu, hipStream_t stream) {
  const dim3 grid(unsigned(a.blocks)), block(kMfNT);
  if (mu == 8)
    hipLaunchKernelGGL((k_gemm_mfma<BP, 8, D, R2>), grid, block, 0, stream, a);
  else if (mu == 4)
    hipLaunchKernelGGL((k_gemm_mfma<BP, 4, D, R2>), grid, block, 0, stream, a);
  else
    return false;
  if constexpr (R2) launch_reduce_split(a, BP, kMfR, stream);
  return true;
}

}  // namespace

bool launch_gemm_mfma(const GemmArgs& a, int bpad, int mu, int depth, bool reduce2, hipStream_t stream) {
  if (reduce2 && depth == 2) {   // split tiles reduced by a second kernel (depth 2 only)
    switch (bpad) {
      case 4: return launch_mfma_bp<4, 2, true>(a, mu, stream);
      case 8: return launch_mfma_bp<8, 2, true>(a, mu, stream);
      case 16: return launch_mfma_bp<16, 2, true>(a, mu, stream);
    }
    return false;
  }
  // 16 batch rows hold 16 more registers per unit in flight: two units ahead (three would spill)
  if (depth == 3 && bpad != 16) {
    switch (bpad) {
      case 4: return launch_mfma_bp<4, 3, false>(a, mu, stream);
      case 8: return launch_mfma_bp<8, 3, false>(a, mu, stream);
    }
  } else if (depth == 2 || depth == 3) {
    switch (bpad) {
      case 4: return launch_mfma_bp<4, 2, false>(a, mu, stream);
      case 8: return launch_mfma_bp<8, 2, false>(a, mu, stream);
      case 16: return launch_mfma_bp<16, 2, false>(a, mu, stream);
    }
  }
  return false;
}

}  // namespace fluxbin
