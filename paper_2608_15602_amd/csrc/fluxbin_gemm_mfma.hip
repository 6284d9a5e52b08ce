// Small-batch (B = 2..32) product of libfluxbin on the gfx950 matrix cores (MFMA).
//
// What is computed is the same as the LUT kernels (Eqs. 10-11 and 15), for every batch row b < B:
//   y[b, i] = sum_c rscale[plane(c)][i] * sum_{v in chunk c} s(i, v) * colscale[v] * x[b, xidx[v]],
// s(i, v) = +1 for a set sign bit and -1 for a clear one. The LUT kernels form the inner sum by table lookups, whose
// cost grows with the batch (one table entry read and added per batch row and sub-vector). With B > 1 the same inner
// sums are a dense contraction over the virtual columns: a (rows x 128) block of signed column scales times a
// (128 x B) block of activations. Here every 32 columns of that contraction are one v_mfma_f32_16x16x32_f16, and the
// cost per sign bit is the same for any B <= 16 (the batch occupies the 16 columns of the MFMA tile). With 17..32 rows
// each decoded operand feeds two MFMA tiles (batch rows 0..15 and 16..31): the decode per sign bit is paid once for
// twice the rows.
//
// Exactness. The A operand is -s(i, v) * colscale[v], an fp16 value (the column scale with its sign bit flipped where
// the sign bit is set), and the B operand is x[b, xidx[v]], also fp16. Their products are exact in the fp32
// accumulation of the matrix core, as x * colscale is exact in fp32 for the LUT kernels (two 11-bit significands). The
// row scale multiplies each 128-column chunk's fp32 sum once (Eq. 15's order), negated, and y is the fp32 sum over
// chunks. Padding columns have column scale 0 and stage x = 0, so they add exactly zero.
//
// Sign decode. By the packed format, row i's 16-byte entry of a chunk holds the chunk's 128 sign bits rotated left by
// R(i) bits (mu = 8: R = 8 (i mod 16); mu = 4: R = 4 (i mod 32)). Lane (r, g) of a 16-row MFMA block needs canonical
// bits 32g .. 32g+31 of its row r: two 32-bit words of the entry and one funnel shift give them, whatever the
// rotation. The K dimension of the contraction is ordered so that element pair k of K step q holds canonical columns
// (32g + 4q + k, 32g + 4q + k + 16): a left shift of the 32 bits by 15 - (4q + k) puts both sign bits at bit
// positions 15 and 31, the fp16 sign bits of the pair, so one three-input bit operation (v_bitop3_b32: and with the
// sign-bit mask, xor with the column-scale pair) forms the operand. The words of two row blocks are shifted together as
// one 64-bit value.
//
// Work decomposition (as in the LUT kernels): a tile is 256 rows, 64 per wavefront of a 256-thread workgroup (four
// 16-row MFMA blocks); a unit is a tile times a super-chunk (256 virtual columns, both stored chunk slots); units are
// numbered tile-major, split into contiguous equal ranges, one per workgroup; split tiles are reduced by the
// deterministic counter protocol of fluxbin_device.h (same partial-sum layout, so its reduction code is shared).
//
// Memory pipeline. Each lane requests its row's whole 16-byte entries of a unit (one 16-byte load per chunk) and one
// 32-bit word of row scales, D units ahead of the unit being multiplied (2 KB of signs per wavefront per unit, no
// byte requested twice); a wavefront passes the entries to its MFMA lanes through its own LDS scratch.
// Activations. The B operands of a super-chunk (x gathered through the VCM index table, in the order the MFMA lanes
// read them, as fp16 pairs) and its signed column-scale pairs do not depend on the row tile. Up to 8 batch rows each
// thread gathers its column pair of a unit itself, with the unit's signs, and writes it to the double-buffered LDS
// staging area one unit ahead. With 16 and 32 rows those gathers would hold 48 or 96 registers of loads in flight,
// so a first kernel (k_mf_image) writes the activations once per call, for every super-chunk, to an image in the
// workspace laid out exactly like the LDS staging area of one unit. The multiplying kernel copies a unit's image into its double-buffered staging
// area with LDS-direct loads (global_load_lds_dwordx4: 16 bytes per lane written straight to LDS, no registers), one
// unit ahead, issued before that step's sign requests. Vector memory operations complete in issue order, so waiting
// until at most the three sign and row-scale requests issued after the copy are outstanding (s_waitcnt vmcnt(3)),
// before the step's barrier, means the copy has landed while the later sign requests stay in flight. The copies are
// written as instructions because the compiler, seeing an LDS-direct load in flight, drains every outstanding load
// before each barrier, which would leave no sign request in flight across the steps.
#include <hip/hip_runtime.h>

#include "fluxbin_device.h"

namespace fluxbin {

namespace {

typedef _Float16 mf_half8 __attribute__((ext_vector_type(8)));
typedef float mf_float4 __attribute__((ext_vector_type(4)));
typedef unsigned int mf_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short mf_u16x2 __attribute__((ext_vector_type(2)));

constexpr int kMfNT = 256;                          // threads per workgroup: four wavefronts of 64 rows
constexpr int kMfR = 256;                           // rows per tile
// Batch rows per MFMA tile is 16; BP = 32 runs two batch tiles against each decoded sign operand.
template <int BP> constexpr int mf_nbt() { return BP > 16 ? BP / 16 : 1; }
// dwords per (chunk, column group, K step) block of staged activation pairs: 16 * mf_nbt rows x 4 pairs + 4 pad
template <int BP> constexpr int mf_xunit() { return 2 * 4 * 4 * mf_xstride(BP); }   // dwords per unit
constexpr int kMfAUnit = 2 * 4 * 16;                // dwords of column-scale pairs per unit
constexpr int kMfScr = 2 * 64 * 4;                  // dwords of a wavefront's sign scratch: 2 chunks x 64 rows x 16 bytes
constexpr int kMfScrUnit = kMfScr + 64;             // dwords of one unit's sign scratch and 64 words of row scales
constexpr int kMfScrWave = 2 * kMfScrUnit;          // dwords of a wavefront's scratch: two units (double buffer)
constexpr int kMfTStride = 68;                      // dwords per batch row of a wavefront's tile-end transpose
constexpr int kMfTRows = 8;                         // batch rows per pass of the transpose (in one unit's scratch)
static_assert(kMfTRows * kMfTStride <= kMfScrUnit, "transpose pass larger than a unit's scratch");

// dwords of a unit's activation image: the staged activation pairs, then the column-scale pairs; a whole number of
// 1 KB LDS-direct requests (64 lanes x 16 bytes)
template <int BP> constexpr int mf_img() { return mf_image_dwords(BP); }
static_assert(mf_img<4>() >= mf_xunit<4>() + kMfAUnit && mf_img<16>() == mf_xunit<16>() + kMfAUnit &&
              mf_img<32>() == mf_xunit<32>() + kMfAUnit, "image smaller than the staging area");

// Activation staging: up to 8 batch rows each thread gathers its column pair of a unit itself (few rows: the loads
// are cheap and a separate image kernel would cost more than it saves); 16 and 32 rows copy the unit's image.
template <int BP> constexpr bool mf_gather() { return BP <= 8; }

// Requested data of one unit: the lane's row entries of both chunks (lane l: row 16 (l >> 4) + (l & 15) of the
// wavefront's 64 rows) and one word of row scales (lane l: rows 2 (l & 31) and 2 (l & 31) + 1 of chunk l >> 5);
// gathering: also the thread's staged column pair, the metadata of its two columns and their x in its half of the
// batch rows.
template <int BP, bool G = mf_gather<BP>()>
struct MfUnitRegs {
  mf_u32x4 e[2];
  uint32_t r;
};
template <int BP>
struct MfUnitRegs<BP, true> {
  mf_u32x4 e[2];
  uint32_t r;
  uint32_t meta[2];     // xidx | colscale << 16 of the thread's columns c and c + 16 (see mf_pair_col)
  uint16_t xv[BP];      // x bits: xv[2i], xv[2i + 1] = columns c, c + 16 of batch row BP/2 * half + i (rows >= B: row B-1)
};

// Buffer resources of a gathering thread's BP/2 batch rows of x, each of range the row's N columns (empty when
// copying images).
template <int BP, bool G = mf_gather<BP>()>
struct MfXRows {};
template <int BP>
struct MfXRows<BP, true> {
  __amdgpu_buffer_rsrc_t r[BP / 2];
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

// Staging ownership when gathering: thread t stages the column pair p = t & 127 of a unit, virtual columns
// c = 32 (p >> 4) + (p & 15) and c + 16 (chunk c >> 7; the pair is one fp16 pair of the MFMA operands), for half t >> 7
// of the batch rows.
__device__ __forceinline__ int mf_pair_col(int t) { return 32 * ((t & 127) >> 4) + (t & 15); }

// Metadata of the thread's two columns of super-chunk sc, through buffer loads (byte offsets 32-bit: the host checks
// the index tables' size).
__device__ __forceinline__ void mf_load_meta(const GemmArgs& a, int sc, int t, uint32_t (&m)[2]) {
  const __amdgpu_buffer_rsrc_t ri = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.xidx), 0,
                                                                       a.NSC * 512, 0x00020000);
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.colscale), 0,
                                                                       a.NSC * 512, 0x00020000);
  const int voff = 2 * mf_pair_col(t), soff = sc * 512;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t xi = __builtin_amdgcn_raw_buffer_load_b16(ri, voff + 32 * i, soff, 0);
    const uint32_t cs = __builtin_amdgcn_raw_buffer_load_b16(rc, voff + 32 * i, soff, 0);
    m[i] = xi | (cs << 16);
  }
}

// Gathers the thread's activations of a unit into u (u.meta must hold the unit's metadata). A padding column's load
// is given an offset outside every range (2^31), for which the load returns zero without reading memory: x is never
// multiplied there, not even by a zero.
template <int BP>
__device__ __forceinline__ void mf_issue_x(const MfXRows<BP>& rx, MfUnitRegs<BP>& u) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t xi = u.meta[i] & 0xFFFFu;
    const int voff = xi == 0xFFFFu ? int(0x80000000u) : int(2 * xi);
#pragma unroll
    for (int b = 0; b < BP / 2; ++b) u.xv[2 * b + i] = __builtin_amdgcn_raw_buffer_load_b16(rx.r[b], voff, 0, 0);
  }
}

// Writes a gathered unit to its staging buffer: the thread's activation pairs and, for half 0, its column-scale pair
// (with sign), in the order the MFMA operands read them. Batch rows b >= B hold row B-1's values: MFMA output column b
// depends on activation column b only, and columns >= B are never stored.
template <int BP>
__device__ __forceinline__ void mf_stage_write(const MfUnitRegs<BP>& u, uint32_t* sx, uint32_t* sa, int t) {
  const int p = t & 127, hg = p >> 4, j = p & 15, q = j >> 2, k = j & 3, half = t >> 7;
  uint32_t* dst = sx + (hg * 4 + q) * mf_xstride(BP) + k + 4 * (BP / 2) * half;
#pragma unroll
  for (int b = 0; b < BP / 2; ++b) dst[4 * b] = __builtin_bit_cast(uint32_t, mf_u16x2{u.xv[2 * b], u.xv[2 * b + 1]});
  if (half == 0) sa[hg * 16 + j] = (u.meta[0] >> 16) | (u.meta[1] & 0xFFFF0000u);
}

// Requests unit c's sign entries and row scales into u (three vector loads per lane). p0, p1: row-scale planes of the
// unit's two chunks.
template <int BP, int MU>
__device__ __forceinline__ void mf_issue(const GemmArgs& a, const MfCursor& c, int32_t p0, int32_t p1, int wave,
                                         int lane, MfUnitRegs<BP>& u) {
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

// LDS address (bytes) of a pointer into the workgroup's LDS.
__device__ __forceinline__ uint32_t mf_lds_addr(const uint32_t* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const uint32_t*)(p)));
}

// Copies the activation image of super-chunk sc (mf_img<BP>() dwords) into the LDS staging area dst, LDS-direct: the
// image's 1 KB requests are dealt round-robin to the four wavefronts (request r: image dwords 256 r .. 256 r + 255,
// lane l's 16 bytes written at dst + 256 r + 4 l). M0 holds the request's LDS address (one wait state between its
// write and the load). Returns nothing to registers; the caller waits with vmcnt before the data is read.
template <int BP>
__device__ __forceinline__ void mf_issue_image(const GemmArgs& a, int sc, uint32_t* dst, int wave, int lane) {
  constexpr int NI = mf_img<BP>() / 256;
  const uint32_t* src = a.img + int64_t(sc) * mf_img<BP>() + 4 * lane;
#pragma unroll
  for (int i = 0; i < (NI + 3) / 4; ++i) {
    const int r = 4 * i + wave;
    if (r < NI)
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                   :
                   : "s"(mf_lds_addr(dst + 256 * r)), "v"(src + 256 * r)
                   : "memory");
  }
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

// Writes a unit's sign entries and row-scale word (requested by mf_issue) to the wavefront's scratch of that unit:
// chunk h's entries at 256 h dwords, one 16-byte entry per row, rows consecutive, then the 64 row-scale words.
template <int BP>
__device__ __forceinline__ void mf_stage_signs(const MfUnitRegs<BP>& u, uint32_t* scr, int lane) {
  *reinterpret_cast<mf_u32x4*>(scr + lane * 4) = u.e[0];
  *reinterpret_cast<mf_u32x4*>(scr + 256 + lane * 4) = u.e[1];
  scr[kMfScr + lane] = u.r;
}

// Multiplies one staged unit into the accumulators of its NBT 16-row batch tiles. xs/as: the unit's staged activation
// (batch tile bt at 64 bt dwords of each block) and column-scale pairs. With BP < 16 a block holds BP rows, and lanes
// of MFMA batch columns >= BP read the next block's dwords: those columns of the product are never stored, and each
// column of an MFMA result depends on that column of its B operand only.
// scr: the wavefront's scratch of the unit (mf_stage_signs). wa[par][c]: dword offset, within a chunk's entries, of
// word c of the two a lane reads from its row of block 0 (row blocks of parity par; block rb adds 64 rb). Reading the
// words separately, with the index wrapped within the entry, needs no copy of an entry's first words after it, and
// the 64 lanes of one read hit 64 different banks: lane (r, g) reads bank 4r + (its word index), and the word indices
// of one r are a permutation of 0..3 over g.
template <int BP, int NBT = mf_nbt<BP>()>
__device__ __forceinline__ void mf_unit(const uint32_t* xs, const uint32_t* as, const uint32_t* scr, int r16, int g,
                                        const uint32_t (&wa)[2][2], uint32_t sh, float (&acc)[NBT][4][4]) {
  constexpr int XS = mf_xstride(BP);
  const uint32_t* srs = scr + kMfScr;
  uint32_t w[2][4];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
      w[h][rb] = __builtin_amdgcn_alignbit(scr[256 * h + 64 * rb + wa[rb & 1][1]],
                                           scr[256 * h + 64 * rb + wa[rb & 1][0]], sh);
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint2 rs[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) rs[rb] = *reinterpret_cast<const uint2*>(srs + h * 32 + 8 * rb + 2 * g);
    // the words of row blocks 2rp and 2rp + 1 as one 64-bit value (high: 2rp + 1), shifted together below
    const uint64_t w2[2] = {(uint64_t(w[h][1]) << 32) | w[h][0], (uint64_t(w[h][3]) << 32) | w[h][2]};
    if constexpr (NBT > 1) {
      // two batch tiles: one pair of row blocks at a time (half the live partial products, the activation and
      // column-scale rows read once per pair), which keeps the kernel within three waves per SIMD
#pragma unroll
      for (int rp = 0; rp < 2; ++rp) {
        mf_float4 tmp[NBT][2];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const mf_u32x4 ac = *reinterpret_cast<const mf_u32x4*>(as + (h * 4 + g) * 16 + 4 * q);
          mf_u32x4 bx[NBT];
#pragma unroll
          for (int bt = 0; bt < NBT; ++bt)
            bx[bt] = *reinterpret_cast<const mf_u32x4*>(xs + ((h * 4 + g) * 4 + q) * XS + 64 * bt + 4 * r16);
          mf_u32x4 av0, av1;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const uint64_t sft = mf_shl64(w2[rp], uint32_t(15 - (4 * q + k)));
            av0[k] = (uint32_t(sft) & 0x80008000u) ^ ac[k];
            av1[k] = (uint32_t(sft >> 32) & 0x80008000u) ^ ac[k];
          }
#pragma unroll
          for (int bt = 0; bt < NBT; ++bt) {
            const mf_float4 c0 = q == 0 ? mf_float4{0.f, 0.f, 0.f, 0.f} : tmp[bt][0];
            const mf_float4 c1 = q == 0 ? mf_float4{0.f, 0.f, 0.f, 0.f} : tmp[bt][1];
            tmp[bt][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mf_half8, av0),
                                                                __builtin_bit_cast(mf_half8, bx[bt]), c0, 0, 0, 0);
            tmp[bt][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mf_half8, av1),
                                                                __builtin_bit_cast(mf_half8, bx[bt]), c1, 0, 0, 0);
          }
        }
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt)
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            const int rb = 2 * rp + i;
            acc[bt][rb][0] = fmaf(-h2f(uint16_t(rs[rb].x)), tmp[bt][i][0], acc[bt][rb][0]);
            acc[bt][rb][1] = fmaf(-h2f(uint16_t(rs[rb].x >> 16)), tmp[bt][i][1], acc[bt][rb][1]);
            acc[bt][rb][2] = fmaf(-h2f(uint16_t(rs[rb].y)), tmp[bt][i][2], acc[bt][rb][2]);
            acc[bt][rb][3] = fmaf(-h2f(uint16_t(rs[rb].y >> 16)), tmp[bt][i][3], acc[bt][rb][3]);
          }
      }
      continue;
    }
    mf_float4 tmp[NBT][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const mf_u32x4 ac = *reinterpret_cast<const mf_u32x4*>(as + (h * 4 + g) * 16 + 4 * q);
      mf_u32x4 bx[NBT];
#pragma unroll
      for (int bt = 0; bt < NBT; ++bt)
        bx[bt] = *reinterpret_cast<const mf_u32x4*>(xs + ((h * 4 + g) * 4 + q) * XS + 64 * bt + 4 * r16);
#pragma unroll
      for (int rp = 0; rp < 2; ++rp) {
        mf_u32x4 av0, av1;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint64_t sft = mf_shl64(w2[rp], uint32_t(15 - (4 * q + k)));
          av0[k] = (uint32_t(sft) & 0x80008000u) ^ ac[k];
          av1[k] = (uint32_t(sft >> 32) & 0x80008000u) ^ ac[k];
        }
        // the decoded operands serve every batch tile
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) {
          const mf_float4 c0 = q == 0 ? mf_float4{0.f, 0.f, 0.f, 0.f} : tmp[bt][2 * rp];
          const mf_float4 c1 = q == 0 ? mf_float4{0.f, 0.f, 0.f, 0.f} : tmp[bt][2 * rp + 1];
          tmp[bt][2 * rp] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mf_half8, av0),
                                                                   __builtin_bit_cast(mf_half8, bx[bt]), c0, 0, 0, 0);
          tmp[bt][2 * rp + 1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
              __builtin_bit_cast(mf_half8, av1), __builtin_bit_cast(mf_half8, bx[bt]), c1, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt)
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        acc[bt][rb][0] = fmaf(-h2f(uint16_t(rs[rb].x)), tmp[bt][rb][0], acc[bt][rb][0]);
        acc[bt][rb][1] = fmaf(-h2f(uint16_t(rs[rb].x >> 16)), tmp[bt][rb][1], acc[bt][rb][1]);
        acc[bt][rb][2] = fmaf(-h2f(uint16_t(rs[rb].y)), tmp[bt][rb][2], acc[bt][rb][2]);
        acc[bt][rb][3] = fmaf(-h2f(uint16_t(rs[rb].y >> 16)), tmp[bt][rb][3], acc[bt][rb][3]);
      }
  }
}

// End of a tile's contribution: y for a tile only this workgroup covers, else its partial sums (slot 0 for the
// workgroup's first tile, 1 for its last), in the layout reduce_tile reads: element (b, row in tile) at b * R + row.
// Lane (b = r16, g) holds rows 16 rb + 4 g + v of the wavefront's 64; the wavefront first transposes them through the
// scratch of the unit it has just multiplied (row block rb of batch row b at (b mod 8) * kMfTStride + 16 rb, eight
// batch rows per pass), so that every store instruction writes 64 consecutive rows of one batch row (whole memory
// lines: scattered 4-byte stores wrote each line several times).
template <int BP>
__device__ __forceinline__ void mf_tile_end(const GemmArgs& a, int tile, bool shared, int slot, int wave, int lane,
                                            int r16, int g, const float (&acc)[mf_nbt<BP>()][4][4], uint32_t* scr) {
  constexpr int TB = BP < kMfTRows ? BP : kMfTRows;
  float* t = reinterpret_cast<float*>(scr);
  float* mine = a.partials + ((int64_t(blockIdx.x) * 2 + slot) * BP) * kMfR + wave * 64 + lane;
  const int64_t row = int64_t(tile) * kMfR + wave * 64 + lane;
#pragma unroll
  for (int b0 = 0; b0 < BP; b0 += TB) {
    constexpr int NBT = mf_nbt<BP>();
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) {   // batch row 16 bt + r16 of the lane's accumulators
      const int b = 16 * bt + r16;
      if ((16 * bt + 16 > b0 && 16 * bt < b0 + TB) && b >= b0 && b < b0 + TB) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
          *reinterpret_cast<mf_float4*>(t + (b - b0) * kMfTStride + 16 * rb + 4 * g) =
              mf_float4{acc[bt][rb][0], acc[bt][rb][1], acc[bt][rb][2], acc[bt][rb][3]};
      }
    }
    if (shared) {
#pragma unroll
      for (int b = b0; b < b0 + TB; ++b)
        __hip_atomic_store(mine + b * kMfR, t[(b - b0) * kMfTStride + lane], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    } else if (row < a.M) {
#pragma unroll
      for (int b = b0; b < b0 + TB; ++b)
        if (b < a.B) store_y(a, b, row, t[(b - b0) * kMfTStride + lane]);
    }
  }
}

template <int BP, int MU, int D>
struct MfKernel {
  static constexpr int IMG = mf_img<BP>();
  struct State {
    int n;
    int first_tile, last_tile;
    bool first_shared, last_shared;
    int n_pending;
    MfCursor cur;    // unit K
    MfCursor nxt;    // unit K + D (clamped to the last unit of the range)
    int img_sc;      // copying images: super-chunk of unit K + 1, whose activation image is copied next
    int stg_sc;      // gathering: super-chunk of unit K + D + 1 (clamped), whose metadata is requested next
    float acc[mf_nbt<BP>()][4][4];
  };

  struct Lane {
    int t, lane, wave, r16, g;
    uint32_t wa[2][2];   // scratch offsets of the two words holding the lane's canonical bits (see mf_unit)
    uint32_t sh;      // funnel shift
  };

  // Unit K of the workgroup (compile-time K < kMfMaxUnits; the launch plan keeps the range within that), with
  // register set K mod (D + 1). Fully unrolled, so no loads are carried through a loop header.
  // Order: copy unit K+1's activation image into its staging buffer (free: unit K-1, its last reader, ended at the
  // previous barrier); request unit K+D's signs and row scales; stage unit K+1's signs and row scales (requested D-1
  // units ago) to the wavefront's scratch of K+1, so that their registers are free during the multiplication; multiply
  // unit K; end a tile (transposing through unit K's scratch, now read); wait for this step's image copy, then meet at
  // the barrier.
  // Gathering: request unit K+D's activations (metadata requested one unit earlier), signs and row scales, and the
  // metadata of unit K+D+1; stage unit K+1's activations, signs and row scales (requested D-1 units ago); multiply unit
  // K; end a tile; meet at the barrier.
  template <int K>
  __device__ static __forceinline__ void step(const GemmArgs& a, State& s, MfUnitRegs<BP> (&ur)[D + 1],
                                              uint32_t (&meta_next)[2], const int* s_planes, uint32_t* ubuf,
                                              uint32_t* scr, const Lane& ln, const MfXRows<BP>& rx) {
    if constexpr (K < kMfMaxUnits) {
      if (K >= s.n) return;
      constexpr int PN = (K + D) % (D + 1);
      constexpr int PS = (K + 1) % (D + 1);
      if constexpr (mf_gather<BP>()) {
        const int kd = K + D < s.n ? K + D : s.n - 1;
        ur[PN].meta[0] = meta_next[0];
        ur[PN].meta[1] = meta_next[1];
        mf_issue_x<BP>(rx, ur[PN]);
        mf_issue<BP, MU>(a, s.nxt, s_planes[2 * kd], s_planes[2 * kd + 1], ln.wave, ln.lane, ur[PN]);
        mf_load_meta(a, s.stg_sc, ln.t, meta_next);
        if (K + D + 1 < s.n) mf_advance(a, s.nxt);
        if (K + D + 2 < s.n && ++s.stg_sc == a.steps) s.stg_sc = 0;
        __builtin_amdgcn_sched_barrier(0);
        if (K + 1 < s.n) {
          uint32_t* nb = ubuf + ((K + 1) & 1) * IMG;
          mf_stage_write<BP>(ur[PS], nb, nb + mf_xunit<BP>(), ln.t);
          mf_stage_signs<BP>(ur[PS], scr + ((K + 1) & 1) * kMfScrUnit, ln.lane);
        }
      } else {
        if (K + 1 < s.n) {
          mf_issue_image<BP>(a, s.img_sc, ubuf + ((K + 1) & 1) * IMG, ln.wave, ln.lane);
          if (++s.img_sc == a.steps) s.img_sc = 0;
        }
        __builtin_amdgcn_sched_barrier(0);
        {
          const int kd = K + D < s.n ? K + D : s.n - 1;
          mf_issue<BP, MU>(a, s.nxt, s_planes[2 * kd], s_planes[2 * kd + 1], ln.wave, ln.lane, ur[PN]);
          if (K + D + 1 < s.n) mf_advance(a, s.nxt);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (K + 1 < s.n) mf_stage_signs<BP>(ur[PS], scr + ((K + 1) & 1) * kMfScrUnit, ln.lane);
      }
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t* ub = ubuf + (K & 1) * IMG;
      mf_unit<BP>(ub, ub + mf_xunit<BP>(), scr + (K & 1) * kMfScrUnit, ln.r16, ln.g, ln.wa, ln.sh, s.acc);
      if (s.cur.sc == a.steps - 1 || K + 1 == s.n) {
        const int tile = s.cur.tile;
        const bool shared = tile == s.first_tile ? s.first_shared : (tile == s.last_tile && s.last_shared);
        mf_tile_end<BP>(a, tile, shared, tile == s.first_tile ? 0 : 1, ln.wave, ln.lane, ln.r16, ln.g, s.acc,
                        scr + (K & 1) * kMfScrUnit);
        if (shared) ++s.n_pending;
#pragma unroll
        for (int bt = 0; bt < mf_nbt<BP>(); ++bt)
#pragma unroll
          for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int v = 0; v < 4; ++v) s.acc[bt][rb][v] = 0.f;
      }
      mf_advance(a, s.cur);
      // copying images: every vector memory operation but the last three (unit K+D's sign and row-scale requests, or
      // tile-end stores issued after them) has completed, so this step's image copy has landed
      if constexpr (!mf_gather<BP>()) asm volatile("s_waitcnt vmcnt(3)" ::: "memory");
      __syncthreads();
      step<K + 1>(a, s, ur, meta_next, s_planes, ubuf, scr, ln, rx);
    }
  }
};

// Activation images of every super-chunk for one call (the first of the two kernels; grid IMG / 256 x NSC): image dword
// d of super-chunk sc is what the staging area of a unit of sc holds at d. Activation part (d < mf_xunit): block
// (h g, q) = d / XS, offset o = d mod XS; o < 4 BP is batch row o / 4, pair k = o mod 4 of K step q: the fp16 pair
// (x[row][xidx[v]], x[row][xidx[v + 16]]) of virtual column v = 256 sc + 32 (h g) + 4 q + k, zero for a column with no
// source or a row >= B; padding dwords are zero. Column-scale part: dword 16 (h g) + j holds the signed column scales
// of columns 32 (h g) + j and that + 16.
template <int BP>
__global__ void __launch_bounds__(256) k_mf_image(GemmArgs a) {
  constexpr int XS = mf_xstride(BP);
  constexpr int XU = 2 * 4 * 4 * XS;
  constexpr int IMG = mf_img<BP>();
  const int sc = blockIdx.y;
  const int d = blockIdx.x * 256 + threadIdx.x;
  const int64_t v0 = int64_t(sc) * 256;
  uint32_t v = 0u;
  if (d < XU) {
    const int blk = d / XS;
    const int o = d - blk * XS;
    const int row = o >> 2;
    if (o < 4 * BP && row < a.B) {
      const int c = 32 * (blk >> 2) + 4 * (blk & 3) + (o & 3);
      const uint32_t i0 = a.xidx[v0 + c], i1 = a.xidx[v0 + c + 16];
      const uint16_t* xr = a.x + int64_t(row) * a.ldx;
      const uint32_t x0 = i0 == 0xFFFFu ? 0u : xr[i0];
      const uint32_t x1 = i1 == 0xFFFFu ? 0u : xr[i1];
      v = x0 | (x1 << 16);
    }
  } else if (d < XU + kMfAUnit) {
    const int e = d - XU;
    const int c = 32 * (e >> 4) + (e & 15);
    v = uint32_t(a.colscale[v0 + c]) | (uint32_t(a.colscale[v0 + c + 16]) << 16);
  }
  a.img[int64_t(sc) * IMG + d] = v;
}

template <int BP, int MU, int D, bool R2>
__global__ void __launch_bounds__(kMfNT, mf_gather<BP>() ? ((BP <= 4 && D == 2 && R2) ? 4 : 3) : (BP > 16 ? 3 : 4))
    k_gemm_mfma(GemmArgs a) {
  using K = MfKernel<BP, MU, D>;
  __shared__ __attribute__((aligned(16))) uint32_t ubuf[2 * K::IMG];
  __shared__ __attribute__((aligned(16))) uint32_t scr_all[4 * kMfScrWave];
  __shared__ int s_planes[2 * kMfMaxUnits];
  __shared__ int s_flag;

  typename K::Lane ln;
  ln.t = threadIdx.x;
  ln.lane = ln.t & 63;
  ln.wave = __builtin_amdgcn_readfirstlane(ln.t >> 6);
  ln.r16 = ln.lane & 15;
  ln.g = ln.lane >> 4;
  // Words of a row's entry that hold canonical bits 32g..32g+31: they start at stored bit (32g - R) mod 128;
  // mu = 4: index 1 for odd row blocks (rows with i mod 32 >= 16 rotate by 64 more bits).
  {
    const int rot0 = MU == 8 ? 8 * ln.r16 : 4 * ln.r16;
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const uint32_t aw = uint32_t(((32 * ln.g - rot0 - (MU == 4 ? 64 * par : 0)) & 127) >> 5);
      ln.wa[par][0] = uint32_t(4 * ln.r16) + aw;
      ln.wa[par][1] = uint32_t(4 * ln.r16) + ((aw + 1) & 3u);
    }
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
  for (int bt = 0; bt < mf_nbt<BP>(); ++bt)
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
      for (int v = 0; v < 4; ++v) s.acc[bt][rb][v] = 0.f;

  // Row-scale planes of the range's chunks (the launch plan keeps n <= kMfMaxUnits).
  if (ln.t < 2 * s.n) {
    int sc = s.cur.sc + (ln.t >> 1);
    while (sc >= a.steps) sc -= a.steps;
    s_planes[ln.t] = a.chunk_plane[2 * sc + (ln.t & 1)];
  }
  MfUnitRegs<BP> ur[D + 1];
  uint32_t meta_next[2];
  MfXRows<BP> rx;
  s.nxt = s.cur;
  if constexpr (mf_gather<BP>()) {
    // the thread's batch rows of x: half t >> 7 of the padded batch (wave-uniform; rows >= B read row B-1)
    const int half = __builtin_amdgcn_readfirstlane(ln.t >> 7);
#pragma unroll
    for (int i = 0; i < BP / 2; ++i) {
      const int b = (BP / 2) * half + i;
      rx.r[i] = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.x + int64_t(b < a.B ? b : a.B - 1) * a.ldx),
                                                  0, 2 * a.N, 0x00020000);
    }
    // metadata of units 0..D
    int sc = s.cur.sc;
#pragma unroll
    for (int k = 0; k <= D; ++k) {
      mf_load_meta(a, sc, ln.t, k < D ? ur[k].meta : meta_next);
      if (k + 1 < s.n && ++sc == a.steps) sc = 0;
    }
    s.stg_sc = sc;   // unit D + 1 (clamped)
    __syncthreads();   // planes in LDS
#pragma unroll
    for (int k = 0; k < D; ++k) {
      const int kk = k < s.n ? k : s.n - 1;
      mf_issue_x<BP>(rx, ur[k]);
      mf_issue<BP, MU>(a, s.nxt, s_planes[2 * kk], s_planes[2 * kk + 1], ln.wave, ln.lane, ur[k]);
      if (k + 1 < s.n) mf_advance(a, s.nxt);
    }
    mf_stage_write<BP>(ur[0], ubuf, ubuf + mf_xunit<BP>(), ln.t);
    mf_stage_signs<BP>(ur[0], scr, ln.lane);
  } else {
    __syncthreads();   // planes in LDS
    // unit 0's image, then the signs and row scales of units 0..D-1
    mf_issue_image<BP>(a, s.cur.sc, ubuf, ln.wave, ln.lane);
    s.img_sc = s.cur.sc + 1 == a.steps ? 0 : s.cur.sc + 1;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < D; ++k) {
      const int kk = k < s.n ? k : s.n - 1;
      mf_issue<BP, MU>(a, s.nxt, s_planes[2 * kk], s_planes[2 * kk + 1], ln.wave, ln.lane, ur[k]);
      if (k + 1 < s.n) mf_advance(a, s.nxt);
    }
    __builtin_amdgcn_sched_barrier(0);
    mf_stage_signs<BP>(ur[0], scr, ln.lane);
    // units 0..D-1 requested after the image: all but their last three requests complete means the image has landed
    asm volatile("s_waitcnt vmcnt(3)" ::: "memory");
  }
  __syncthreads();
  K::template step<0>(a, s, ur, meta_next, s_planes, ubuf, scr, ln, rx);
  if constexpr (!R2) {
    const int pend0 = s.first_shared ? s.first_tile : s.last_tile;
    publish_pending<kMfNT, 1, BP>(a, pend0, s.last_tile, s.n_pending, &s_flag);
  }
}

template <int BP, int D, bool R2>
bool launch_mfma_bp(const GemmArgs& a, int mu, hipStream_t stream) {
  if (mu != 8 && mu != 4) return false;
  if constexpr (!mf_gather<BP>())
    hipLaunchKernelGGL((k_mf_image<BP>), dim3(unsigned(mf_img<BP>() / 256), unsigned(a.NSC)), dim3(256), 0, stream,
                       a);
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
      case 32: return launch_mfma_bp<32, 2, true>(a, mu, stream);
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
