// Batch-1 LUT-GEMV of libfluxbin for layers with few rows (the product of Eqs. 10-15, as the batch-1 kernel in
// fluxbin_gemv.hip computes it): row-complete workgroups, so that no partial sum crosses a workgroup.
//
// Why a second batch-1 kernel. A layer of a few thousand rows carries a few MB of sign data, and spread over the
// chip that is a handful of units per CU. There the split-tile kernel spends most of a call outside its steady state:
// its start-up, then the cross-workgroup reduction of split tiles (partial-sum stores, a counter round trip, the
// reducer's loads and the y stores), each a dependent round trip to memory. Here a workgroup owns 16 rows and every
// super-chunk of them: its W wavefronts take every W-th super-chunk, build that unit's tables, look them up, and add
// their partial sums through LDS in a fixed order at the end. The tables of a unit are built once per workgroup
// instead of once per tile of 512-1024 rows; with mu = 4 tables that redundancy costs 20 adds and 16 LDS writes per
// lane and unit.
//
// Tables. mu = 4 patterns for either packed mu (a mu = 8 sub-vector byte is two mu = 4 nibbles, and both packed
// rotations move whole nibbles). Per unit 64 tables, one per (chunk h, canonical nibble s), of 16 fp32 entries, one
// table built by each of the wavefront's 64 lanes: T[e] = sum_n xv[n] (2 bit_n(e) - 1) over the nibble's four folded
// activations xv = x[xidx] * colscale (exact in fp32, Eq. 11; VCM gather through the index table, Eq. 13), formed as
// (+-xv0 +-xv1) + (+-xv2 +-xv3). Entry e of table T is LDS float e*64 + T, so the 64 lanes of a table write hit 64
// banks.
//
// Lookups. Lane (r, p) handles row r of the workgroup and dword p of its 16-byte entries: per chunk the eight stored
// nibbles Q = 8p + j, whose canonical nibble is (Q + rot(i)) mod 32 (mu = 8: rot = 2i, and rows with i mod 32 >= 16
// hold the chunk pair swapped; mu = 4: rot = i). The lane sums its eight lookups of a chunk and multiplies the sum by
// the row's scale of that chunk (Eq. 15). Salient chunks with FG = 8 or 16 fine row-scale groups (the paper's s16 /
// s8 configurations at mu = 8) sum their lookups per stored position block and multiply each block's sum by its own
// scale; other fine layouts use the other kernels. The four lanes of a row are then added pairwise (lane xor 1, then xor 2: each addition is commutative, so
// both lanes of a pair hold the same bits), and the W wavefronts' sums in wavefront order.
//
// Activations. The whole x (N <= kRwMaxN fp16) is staged in LDS once per workgroup, one round trip at the start
// that overlaps the first sign requests; every gather then reads LDS.
#include <hip/hip_runtime.h>

#include "fluxbin_device.h"

namespace fluxbin {

namespace {

constexpr int kRwRows = 16;       // output rows per workgroup (kRwSteps, kRwMaxN: fluxbin_internal.h)

// Requested data of one unit for one lane.
typedef unsigned int mf_u32x2_rw __attribute__((ext_vector_type(2)));

template <int FG, int RB>
struct RwRegs {
  uint32_t w[RB][2];    // per row of the lane: dword p of the row's entries of chunks 2sc (w[.][0]) and 2sc + 1
  // fp16 row scales of each row for the two chunks: one (low half of rs[.][h][0]), or for a chunk with FG fine groups
  // the scales of the lane's position blocks (FG = 16: four, FG = 8: two)
  uint32_t rs[RB][2][FG == 16 ? 2 : 1];
  uint2 cs;         // fp16 column scales of the four columns of the lane's table
  uint2 xi;         // their activation indices (0xFFFF: no source)
};

template <int RB>
struct RwLane {
  int t, lane, w, r, p;
  uint32_t row[RB];   // the lane's rows r, r + 16, ... of the workgroup (clamped to Mp - 1; rows >= M are not stored)
  int hb[RB];         // mu = 8: the row holds the chunk pair of a super-chunk swapped
  int tv;             // the lane's table: virtual column of its first column within a super-chunk (0..252)
  int hA;             // chunk of the lane's first eight lookups (rw_lookup)
  uint32_t sh;        // rotation of its sign dwords before the lookups (0 or 4 bits)
  uint32_t colp[4];   // byte k mod 4 of colp[k / 4]: byte offset of the table column of lookup k, (chunk*32 + s)*4
  uint32_t wblk;      // (w << 4) in every byte: the wavefront's table block in bits 12..15 of a lookup address
  uint32_t colf[4];   // the same for chunks with fine row-scale groups (their position rotation, no odd-p shift)
};

// Buffer resources of the packed sections and per-lane byte offsets: every load is a buffer load with the unit's
// offset in a scalar register (the launch plan keeps the sign and row-scale sections below 2^31 bytes).
template <int RB>
struct RwBufs {
  __amdgpu_buffer_rsrc_t signs, rscale, colscale, xidx;
  uint32_t voff_w[RB][2];   // sign dword p of each of the lane's rows in the slot holding chunk 2sc + h, super-chunk 0
  uint32_t voff_rs[RB];     // each of the lane's rows in a row-scale plane
  uint32_t voff_cv;     // the lane's table's four columns in a super-chunk's column tables
};

// Requests a unit's sign dwords, column scales and activation indices (addresses known from the unit alone).
template <int FG, int RB>
__device__ __forceinline__ void rw_issue(const GemmArgs& a, const RwBufs<RB>& bf, int sc, RwRegs<FG, RB>& u) {
  const int soff_w = 2 * sc * a.Mp * 16;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      u.w[rb][h] = __builtin_amdgcn_raw_buffer_load_b32(bf.signs, int(bf.voff_w[rb][h]), soff_w, 0);
  const mf_u32x2_rw cs = __builtin_amdgcn_raw_buffer_load_b64(bf.colscale, int(bf.voff_cv), sc * 512, 0);
  const mf_u32x2_rw xi = __builtin_amdgcn_raw_buffer_load_b64(bf.xidx, int(bf.voff_cv), sc * 512, 0);
  u.cs = make_uint2(cs[0], cs[1]);
  u.xi = make_uint2(xi[0], xi[1]);
}

// Requests a unit's row scales from the planes of its two chunks (wave-uniform). A chunk with FG fine
// groups owns FG planes read as [Mp][FG]: slot b of a row scales its stored position block b (16 / FG positions),
// so the lane's blocks are contiguous: FG = 16 slots 4p..4p+3 (8 bytes), FG = 8 slots 2p, 2p+1 (4 bytes).
template <int FG, int RB>
__device__ __forceinline__ void rw_issue_rs(const GemmArgs& a, const RwBufs<RB>& bf, const int (&planes)[2], bool fine,
                                           int p, RwRegs<FG, RB>& u) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int plane = planes[h];
      if (FG != 0 && fine) {
        const int voff = int(bf.voff_rs[rb]) * FG + (FG == 16 ? 8 : 4) * p;
        if constexpr (FG == 16) {
          const mf_u32x2_rw v = __builtin_amdgcn_raw_buffer_load_b64(bf.rscale, voff, plane * a.Mp * 2, 0);
          u.rs[rb][h][0] = v[0];
          u.rs[rb][h][FG == 16 ? 1 : 0] = v[1];
        } else {
          u.rs[rb][h][0] = __builtin_amdgcn_raw_buffer_load_b32(bf.rscale, voff, plane * a.Mp * 2, 0);
        }
      } else {
        u.rs[rb][h][0] = __builtin_amdgcn_raw_buffer_load_b16(bf.rscale, int(bf.voff_rs[rb]), plane * a.Mp * 2, 0);
      }
    }
  }
}

// Builds the lane's table of a unit into tab (entry e at e*64 + lane).
template <int FG, int RB>
__device__ __forceinline__ void rw_build(const RwRegs<FG, RB>& u, const uint16_t* xl, uint32_t n_x, float* tab,
                                         int lane) {
  float xv[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    const uint32_t xi = ((n < 2 ? u.xi.x : u.xi.y) >> (16 * (n & 1))) & 0xFFFFu;
    const uint32_t cs = ((n < 2 ? u.cs.x : u.cs.y) >> (16 * (n & 1))) & 0xFFFFu;
    const uint16_t xb = xl[xi < n_x ? xi : n_x];   // xl[N] = 0: a column with no source (index 0xFFFF)
    xv[n] = h2f(xb) * h2f(uint16_t(cs));
  }
  // pair sums: lo[e & 3] = +-xv0 +-xv1, hi[e >> 2] = +-xv2 +-xv3 (bit set: +)
  const float s01 = xv[0] + xv[1], d01 = xv[0] - xv[1];
  const float s23 = xv[2] + xv[3], d23 = xv[2] - xv[3];
  const float lo[4] = {-s01, d01, -d01, s01};
  const float hi[4] = {-s23, d23, -d23, s23};
#pragma unroll
  for (int e = 0; e < 16; ++e) tab[e * 64 + lane] = lo[e & 3] + hi[e >> 2];
}

// Looks up a unit for row rb of the lane: the two chunks' sums, each times its row scale, added to acc. Lookup k of the
// lane reads chunk hA (k < 8) or the other (k >= 8), and its dword rotated right by sh bits puts the nibble at bits
// 4 (k mod 8) (see RwLane setup): the 64 lanes of every read then hit 64 different tables, i.e. 64 banks. Units with
// fine row-scale groups keep the stored nibble order (their lookups are summed per position block and each block
// sum is multiplied by its own scale). The lane's second row (RB = 2, mu = 8 only) is 16 rows further: its rotation
// 2i is the same mod 32, so the same table columns; its chunk pair is stored swapped relative to the first row, which
// the row's own sign offsets (voff_w) already account for.
template <int FG, int RB>
__device__ __forceinline__ void rw_lookup_row(const RwRegs<FG, RB>& u, int rb, bool fine, const float* tabs,
                                              const RwLane<RB>& ln, float& acc) {
  const char* tb = reinterpret_cast<const char*>(tabs);
  const uint32_t wa = ln.hA ? u.w[rb][1] : u.w[rb][0], wb = ln.hA ? u.w[rb][0] : u.w[rb][1];
  const bool fu = FG != 0 && fine;
  const uint32_t sh = fu ? 0u : ln.sh;
  const uint32_t w2[2] = {__builtin_amdgcn_alignbit(wa, wa, sh), __builtin_amdgcn_alignbit(wb, wb, sh)};
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    // even and odd nibbles in the low four bits of their bytes, the wavefront's table block (4 KB) in the high four;
    // one v_perm_b32 then forms a lookup's byte address: byte 0 the table column, byte 1 block and pattern
    const uint32_t ev = (w2[c] & 0x0F0F0F0Fu) | ln.wblk, od = ((w2[c] >> 4) & 0x0F0F0F0Fu) | ln.wblk;
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = 8 * c + j;
      const uint32_t sel = 0x0C0C0000u | (uint32_t(4 + (j >> 1)) << 8) | uint32_t(k & 3);
      const uint32_t cols = fu ? ln.colf[k >> 2] : ln.colp[k >> 2];
      v[j] = *reinterpret_cast<const float*>(tb + __builtin_amdgcn_perm((j & 1) ? od : ev, cols, sel));
    }
    const int h = ln.hA ^ c;
    if (fu) {
      // FG = 16: four blocks of two lookups (stored byte 4p + b); FG = 8: two blocks of four
      constexpr int PER = FG == 16 ? 2 : 4;
#pragma unroll
      for (int b = 0; b < 8 / PER; ++b) {
        float sb = v[PER * b];
#pragma unroll
        for (int q = 1; q < PER; ++q) sb += v[PER * b + q];
        constexpr int NW = FG == 16 ? 2 : 1;
        const int wi = FG == 16 ? (b >> 1) : 0;
        const uint32_t word = h ? u.rs[rb][1][wi < NW ? wi : 0] : u.rs[rb][0][wi < NW ? wi : 0];
        acc = fmaf(h2f(uint16_t(word >> (16 * (b & 1)))), sb, acc);
      }
    } else {
      float sum = v[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) sum += v[j];
      acc = fmaf(h2f(uint16_t(h ? u.rs[rb][1][0] : u.rs[rb][0][0])), sum, acc);
    }
  }
}

template <int FG, int RB>
__device__ __forceinline__ void rw_lookup(const RwRegs<FG, RB>& u, bool fine, const float* tabs, const RwLane<RB>& ln,
                                          float (&acc)[RB]) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) rw_lookup_row<FG, RB>(u, rb, fine, tabs, ln, acc[rb]);
}

template <int MU, int W, int D, int FG, int RB>
struct RwKernel {
  // Unit K of the wavefront (super-chunk w + K*W), with register set K mod (D + 1); fully unrolled, so that no load
  // is carried through a loop header.
  template <int K>
  __device__ static __forceinline__ void step(const GemmArgs& a, const RwLane<RB>& ln, const RwBufs<RB>& bf, int n,
                                              RwRegs<FG, RB> (&ur)[D + 1], const int* s_plane, const uint16_t* xl,
                                              float* tab, const float* tabs, float (&acc)[RB]) {
    if constexpr (K < kRwSteps) {
      if (K >= n) return;
      if (K + D < n) {
        RwRegs<FG, RB>& nx = ur[(K + D) % (D + 1)];
        const int scn = ln.w + (K + D) * W;
        rw_issue<FG, RB>(a, bf, scn, nx);
        // planes from LDS (staged in the prologue): no load waits for another
        const int planes[2] = {__builtin_amdgcn_readfirstlane(s_plane[2 * scn]),
                               __builtin_amdgcn_readfirstlane(s_plane[2 * scn + 1])};
        rw_issue_rs<FG, RB>(a, bf, planes, 2 * scn >= a.nfc, ln.p, nx);
      }
      const int sc = ln.w + K * W;
      rw_build<FG, RB>(ur[K % (D + 1)], xl, uint32_t(a.N), tab, ln.lane);
      rw_lookup<FG, RB>(ur[K % (D + 1)], 2 * sc >= a.nfc, tabs, ln, acc);
      step<K + 1>(a, ln, bf, n, ur, s_plane, xl, tab, tabs, acc);
    }
  }
};

// RB > 1: each lane also handles the rows 16, 32 further (16 RB rows per workgroup, the tables of a unit serving RB
// times the rows); mu = 8 only, where those rows' table columns are the first row's: the rotation 2i is the same mod
// 32, and a fine chunk's stored byte order (colf) depends on i mod 16 only.
template <int MU, int W, int D, int FG, int RB>
__global__ void __launch_bounds__(64 * W) k_gemv_rows(GemmArgs a) {
  static_assert(FG == 0 || MU == 8, "fine row-scale groups: mu = 8 only");
  static_assert(RB == 1 || ((RB == 2 || RB == 3) && MU == 8), "several rows per lane: mu = 8");
  constexpr int NT = 64 * W;
  constexpr int ROWS = kRwRows * RB;
  extern __shared__ __attribute__((aligned(16))) uint16_t xl[];   // x: N fp16 (dynamic size, at most kRwMaxN)
  __shared__ __attribute__((aligned(16))) float tabs[W * 16 * 64];
  __shared__ float s_red[W * ROWS];
  __shared__ int s_plane[2 * 8 * kRwSteps];   // row-scale plane of every chunk (NCP <= 2 * 8 * kRwSteps)

  RwLane<RB> ln;
  ln.t = threadIdx.x;
  ln.lane = ln.t & 63;
  ln.w = __builtin_amdgcn_readfirstlane(ln.t >> 6);
  ln.r = ln.lane >> 2;
  ln.p = ln.lane & 3;
  const int row0 = int(blockIdx.x) * ROWS;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    // Mp is a multiple of 64 and row0 < M: with 16 or 32 rows per workgroup every row is below Mp; with 48 the last
    // workgroup's rows past Mp - 1 read row Mp - 1 (same rotation parity, never stored)
    const int r_raw = row0 + ln.r + kRwRows * rb;
    ln.row[rb] = uint32_t(r_raw < a.Mp ? r_raw : a.Mp - 1);
    ln.hb[rb] = MU == 8 ? int((uint32_t(row0 + ln.r + kRwRows * rb) >> 4) & 1u) : 0;
  }
  ln.tv = (ln.lane >> 5) * 128 + 4 * (ln.lane & 31);
  // Lookup order: at lookup k the lane reads chunk h_k = hA ^ (k >= 8) and its stored nibble 8p + j_k, canonical nibble
  // s_k = (8p + j_k + rot) mod 32. mu = 8 (rot = 2i): hA = p >> 1, j_k = (k + (p & 1)) mod 8, so lanes p and p ^ 1 read
  // nibbles of opposite parity and the 32 lanes of a chunk 32 different s; mu = 4 (rot = i): hA = p & 1, j_k = k mod
  // 8, so lanes p and p ^ 2 read s and s + 16. The odd-p shift of j is a rotation of the dword by one nibble.
  {
    const int rot = MU == 8 ? int(2u * ln.row[0]) : int(ln.row[0]);
    ln.hA = MU == 8 ? (ln.p >> 1) : (ln.p & 1);
    const int jo = MU == 8 ? (ln.p & 1) : 0;
    ln.sh = uint32_t(4 * jo);
    ln.wblk = uint32_t(ln.w << 4) * 0x01010101u;
#pragma unroll
    for (int q = 0; q < 4; ++q) ln.colp[q] = 0u;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int h = ln.hA ^ (k >> 3);
      const int j = ((k & 7) + jo) & 7;
      ln.colp[k >> 2] |= uint32_t((h * 32 + ((8 * ln.p + j + rot) & 31)) * 4) << (8 * (k & 3));
    }
    // fine chunks (mu = 8): stored byte q of row i holds sub-vector byte ((q/n + i/n) mod FG) n + ((q mod n) + i) mod n,
    // n = 16 / FG; its low / high nibble is canonical nibble 2u / 2u + 1; nibble order j = k mod 8 (no shift)
#pragma unroll
    for (int q = 0; q < 4; ++q) ln.colf[q] = 0u;
    if constexpr (FG != 0) {
      constexpr int NB = 16 / FG;
      const int i = int(ln.row[0]);
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int h = ln.hA ^ (k >> 3);
        const int j = k & 7;
        const int q = 4 * ln.p + (j >> 1);
        const int u = ((q / NB + i / NB) % FG) * NB + ((q % NB) + i) % NB;
        ln.colf[k >> 2] |= uint32_t((h * 32 + 2 * u + (j & 1)) * 4) << (8 * (k & 3));
      }
    }
  }
  const int n = ln.w < a.NSC ? (a.NSC - 1 - ln.w) / W + 1 : 0;   // super-chunks w, w + W, ...

  // x and the row-scale planes to LDS first: x is a few KB that every workgroup reads (from L2 after the first), and
  // its LDS writes would otherwise wait for the sign requests issued before them (vector loads complete in order)
  if ((reinterpret_cast<uintptr_t>(a.x) & 3u) == 0) {
    const uint32_t* x32 = reinterpret_cast<const uint32_t*>(a.x);
    uint32_t* xl32 = reinterpret_cast<uint32_t*>(xl);
    for (int d = ln.t; d < (a.N >> 1); d += NT) xl32[d] = x32[d];
    if ((a.N & 1) && ln.t == 0) xl[a.N - 1] = a.x[a.N - 1];
  } else {
    for (int d = ln.t; d < a.N; d += NT) xl[d] = a.x[d];
  }
  if (ln.t == 0) xl[a.N] = 0;
  for (int c = ln.t; c < 2 * a.NSC; c += NT) s_plane[c] = a.chunk_plane[c];
  RwBufs<RB> bf;
  bf.signs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(a.signs), 0, a.NCP * a.Mp * 16, 0x00020000);
  bf.rscale = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.rscale), 0, 0x7FFFFFFF, 0x00020000);
  bf.colscale = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.colscale), 0, a.NCP * 256, 0x00020000);
  bf.xidx = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.xidx), 0, a.NCP * 256, 0x00020000);
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int slot = MU == 8 ? (h ^ ln.hb[rb]) : h;
      bf.voff_w[rb][h] = uint32_t(slot * a.Mp * 16) + ln.row[rb] * 16u + 4u * uint32_t(ln.p);
    }
    bf.voff_rs[rb] = ln.row[rb] * 2u;
  }
  bf.voff_cv = uint32_t(ln.tv) * 2u;
  RwRegs<FG, RB> ur[D + 1];
#pragma unroll
  for (int k = 0; k < D; ++k)
    if (k < n) rw_issue<FG, RB>(a, bf, ln.w + k * W, ur[k]);
  // the first units' row scales before the barrier (planes by scalar loads), so that their round trip overlaps the
  // activation staging instead of following it
#pragma unroll
  for (int k = 0; k < D; ++k) {
    if (k < n) {
      const int sc = ln.w + k * W;
      const int planes[2] = {load_uniform_i32(a.chunk_plane, 2 * sc), load_uniform_i32(a.chunk_plane, 2 * sc + 1)};
      rw_issue_rs<FG, RB>(a, bf, planes, 2 * sc >= a.nfc, ln.p, ur[k]);
    }
  }
  __syncthreads();   // x and the planes staged

  float acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = 0.f;
  RwKernel<MU, W, D, FG, RB>::template step<0>(a, ln, bf, n, ur, s_plane, xl, tabs + ln.w * (16 * 64), tabs, acc);

  // each row's four lanes, then the wavefronts in order
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    acc[rb] += __shfl_xor(acc[rb], 1);
    acc[rb] += __shfl_xor(acc[rb], 2);
    if (ln.p == 0) s_red[ln.w * ROWS + ln.r + kRwRows * rb] = acc[rb];
  }
  __syncthreads();
  if (ln.t < ROWS) {
    float y = s_red[ln.t];
#pragma unroll
    for (int w = 1; w < W; ++w) y += s_red[w * ROWS + ln.t];
    const int64_t row = int64_t(row0) + ln.t;
    if (row < a.M) store_y(a, 0, row, y);
  }
}

template <int W, int D>
bool launch_rows_wd(const GemmArgs& a, int mu, int fg, int rb, hipStream_t stream) {
  const dim3 grid(unsigned((a.M + kRwRows * rb - 1) / (kRwRows * rb))), block(64 * W);
  const unsigned xl_bytes = unsigned(((a.N + 1) * 2 + 15) & ~15);   // x and one zero entry
  if (rb == 2 || rb == 3) {   // launch plan: mu = 8, 16 wavefronts, two units ahead
    if constexpr (W == 16 && D == 2) {
      if (mu != 8 || (fg != 0 && fg != 8 && fg != 16)) return false;
      if (rb == 2) {
        if (fg == 0) hipLaunchKernelGGL((k_gemv_rows<8, W, D, 0, 2>), grid, block, xl_bytes, stream, a);
        if (fg == 8) hipLaunchKernelGGL((k_gemv_rows<8, W, D, 8, 2>), grid, block, xl_bytes, stream, a);
        if (fg == 16) hipLaunchKernelGGL((k_gemv_rows<8, W, D, 16, 2>), grid, block, xl_bytes, stream, a);
      } else {
        if (fg == 0) hipLaunchKernelGGL((k_gemv_rows<8, W, D, 0, 3>), grid, block, xl_bytes, stream, a);
        if (fg == 8) hipLaunchKernelGGL((k_gemv_rows<8, W, D, 8, 3>), grid, block, xl_bytes, stream, a);
        if (fg == 16) hipLaunchKernelGGL((k_gemv_rows<8, W, D, 16, 3>), grid, block, xl_bytes, stream, a);
      }
      return true;
    }
    return false;
  }
  if (rb != 1) return false;
  if (mu == 8 && fg == 0)
    hipLaunchKernelGGL((k_gemv_rows<8, W, D, 0, 1>), grid, block, xl_bytes, stream, a);
  else if (mu == 8 && fg == 8)
    hipLaunchKernelGGL((k_gemv_rows<8, W, D, 8, 1>), grid, block, xl_bytes, stream, a);
  else if (mu == 8 && fg == 16)
    hipLaunchKernelGGL((k_gemv_rows<8, W, D, 16, 1>), grid, block, xl_bytes, stream, a);
  else if (mu == 4 && fg == 0)
    hipLaunchKernelGGL((k_gemv_rows<4, W, D, 0, 1>), grid, block, xl_bytes, stream, a);
  else
    return false;
  return true;
}

template <int W>
bool launch_rows_w(const GemmArgs& a, int mu, int depth, int fg, int rb, hipStream_t stream) {
  switch (depth) {
    case 2: return launch_rows_wd<W, 2>(a, mu, fg, rb, stream);
    case 4: return launch_rows_wd<W, 4>(a, mu, fg, rb, stream);
    case 6: return launch_rows_wd<W, 6>(a, mu, fg, rb, stream);
  }
  return false;
}

}  // namespace

bool launch_gemv_rows(const GemmArgs& a, int mu, int waves, int depth, int fg, int rb, hipStream_t stream) {
  if (a.B != 1 || a.N > kRwMaxN || a.NSC > waves * kRwSteps || a.NSC > 8 * kRwSteps) return false;
  switch (waves) {
    case 4: return launch_rows_w<4>(a, mu, depth, fg, rb, stream);
    case 8: return launch_rows_w<8>(a, mu, depth, fg, rb, stream);
    case 16: return launch_rows_w<16>(a, mu, depth, fg, rb, stream);
  }
  return false;
}

}  // namespace fluxbin
