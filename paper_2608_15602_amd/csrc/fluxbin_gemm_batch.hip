// Small-batch (B = 2..16) LUT-GEMM of libfluxbin for gfx950, mu = 8.
//
// What is computed is the same as the batch-1 kernel (Sec. 3.2, Eqs. 11-15) for every batch row b < B:
//   y[b, i] = sum_c rscale[plane(c)][i] * sum_{s < 16} LUT_{b,c,s}[p(i, c, s)],
//   LUT_{b,c,s}[p] = sum_n xv[b, 128c + 8s + n] (2 bit_n(p) - 1),   xv = x[xidx] * colscale.
// Each sign word is read from HBM once and used for every batch row (the tables are what grows with B).
//
// Work decomposition, as in the batch-1 kernel: a tile is 1024 rows (one row per thread of a 1024-thread workgroup);
// a unit is one tile times one super-chunk (two 128-column chunks, i.e. both stored sign slots of a row); units are
// numbered tile-major and split into equal contiguous ranges, one per workgroup; split tiles are reduced by the
// counter protocol of fluxbin_device.h. So the sign stream has the batch-1 kernel's access pattern.
//
// A workgroup handles one group of (up to) four batch rows, blockIdx.y; larger batches launch one row of workgroups
// per group. The groups read the same sign data at nearly the same time, so HBM streams it about once (the 256 MB
// last-level cache serves the repeats), while the table work, which grows with B and bounds this kernel, spreads over
// all CUs. A unit is processed in two sub-steps, one per chunk. LDS holds two table buffers of 256 patterns x 16
// sub-vectors x 4 batch rows (64 KB each; buffer h holds chunk h of a unit): entry (p, s, b) at (p*16 + s)*4 + b, so
// one ds_read_b128 returns the four batch values of a lookup. By the packed format a lane of row i reads sub-vector
// (q + i) mod 16 at byte q, so any 16 consecutive lanes read 16 different sub-vectors, i.e. all 64 LDS banks once:
// the lookups are conflict-free. Each sub-step builds the tables of the next chunk in the other buffer and looks up
// the current one. The folded activations of a unit (256 columns x 4 batch rows, fp32) are staged through a two-slot
// LDS ring: they are requested four units ahead into registers and written two units ahead, so neither wait stalls
// the sign stream.
#include <hip/hip_runtime.h>

#include "fluxbin_device.h"

namespace fluxbin {

struct Bat {
  static constexpr int NT = 1024;
  static constexpr int BPN = 4;               // batch rows staged per workgroup (NB <= BPN of them are computed)
  static constexpr int TBL = 256 * 16 * 4;   // floats per table buffer (64 KB)
  static constexpr int XSS = 12;             // floats per (chunk, batch row, sub-vector) in the staging layout
  static constexpr int XC = BPN * 16 * XSS;  // floats per staged chunk
  static constexpr int XS = 2 * XC;          // floats per staged unit
};

// Per-thread constants of the current tile: byte offsets of the thread's row in the two stored sign slots of a
// super-chunk, and in a row-scale plane.
struct BatRow {
  uint32_t soff0, soff1;   // row * 16 and (Mp + row) * 16 (below 2^32: M <= 2^27)
  uint32_t roff;           // (row >> 1) * 4
};

__device__ __forceinline__ void bat_row_set(const GemmArgs& a, BatRow& rw, int tile) {
  const int row_raw = tile * 1024 + int(threadIdx.x);
  const uint32_t row = uint32_t(row_raw < a.Mp ? row_raw : a.Mp - 1);   // rows past M are never stored
  rw.soff0 = row * 16u;
  rw.soff1 = (uint32_t(a.Mp) + row) * 16u;
  rw.roff = (row >> 1) * 4u;
}

// Request cursor (wave-uniform): the unit (tile, super-chunk sc) requested next. Past the workgroup's range the
// requests continue (so that the number of loads in flight, which the waits count, is the same on every path) from a
// 1 KB region at the start of the sign section and the first row-scale word.
struct BatCursor {
  int tile, sc;
  const uint8_t* sbase;   // signs + sc * 2 * Mp * 16
  bool dummy;
  BatRow rw;
};

__device__ __forceinline__ void bat_cursor_init(const GemmArgs& a, BatCursor& cu, int tile, int sc) {
  cu.tile = tile;
  cu.sc = sc;
  cu.dummy = false;
  cu.sbase = a.signs + int64_t(sc) * 2 * a.Mp * 16;
  bat_row_set(a, cu.rw, tile);
}

__device__ __forceinline__ void bat_cursor_advance(const GemmArgs& a, BatCursor& cu, bool has_next) {
  if (!has_next) {
    cu.dummy = true;
    return;
  }
  if (++cu.sc == a.steps) {
    cu.sc = 0;
    ++cu.tile;
    cu.sbase = a.signs;
    bat_row_set(a, cu.rw, cu.tile);
  } else {
    cu.sbase += int64_t(2) * a.Mp * 16;
  }
}

struct BatRing {
  uint32_t w[8];   // the row's two 16-byte sign entries of the super-chunk (stored slots 0 and 1)
  uint32_t r[2];   // 32-bit words with the fp16 row scales of rows (i & ~1, i | 1) for chunks 2sc and 2sc+1
};

// Loads of the cursor's unit (wave-uniform bases, 32-bit per-lane offsets): both sign entries, and the row-scale
// words of its two chunks from planes pa and pb.
__device__ __forceinline__ void bat_issue_signs(const GemmArgs& a, const BatCursor& cu, BatRing& rg) {
  const uint8_t* sb = cu.dummy ? a.signs : cu.sbase;
  const uint32_t o0 = cu.dummy ? (threadIdx.x & 63u) * 16u : cu.rw.soff0;
  const uint32_t o1 = cu.dummy ? (threadIdx.x & 63u) * 16u : cu.rw.soff1;
  const uint4 v0 = load_stream16(sb + o0);
  const uint4 v1 = load_stream16(sb + o1);
  rg.w[0] = v0.x; rg.w[1] = v0.y; rg.w[2] = v0.z; rg.w[3] = v0.w;
  rg.w[4] = v1.x; rg.w[5] = v1.y; rg.w[6] = v1.z; rg.w[7] = v1.w;
}

__device__ __forceinline__ void bat_issue_rscale(const GemmArgs& a, const BatCursor& cu, int32_t pa, int32_t pb,
                                                 BatRing& rg) {
  const uint32_t ro = cu.dummy ? 0u : cu.rw.roff;
  const uint8_t* ra = reinterpret_cast<const uint8_t*>(a.rscale) + int64_t(pa) * a.Mp * 2;
  const uint8_t* rb = reinterpret_cast<const uint8_t*>(a.rscale) + int64_t(pb) * a.Mp * 2;
  rg.r[0] = *reinterpret_cast<const uint32_t*>(ra + ro);
  rg.r[1] = *reinterpret_cast<const uint32_t*>(rb + ro);
}

// Staging cursor (wave-uniform): unit requested for staging next: its index in the workgroup, super-chunk sc, and
// (2sc) mod ncg for the global-chunk column arithmetic.
struct BatStageCursor {
  int k, sc, cm;
};

__device__ __forceinline__ void bat_stage_cursor_next(const GemmArgs& a, BatStageCursor& s) {
  ++s.k;
  if (++s.sc == a.steps) {
    s.sc = 0;
    s.cm = 0;
  } else {
    s.cm += 2;
    if (s.cm >= a.ncg) s.cm -= a.ncg;
  }
}

// Staging registers of one unit: thread t holds column t & 255 of the unit (chunk 2sc + ((t >> 7) & 1)) for batch
// row t >> 8.
struct BatStage {
  uint32_t xb;   // x bits
  uint32_t cs;   // column scale bits
  bool ok;       // a real activation (else the staged value is 0)
};

// Request the activations of the staging cursor's unit. Global chunks read x[b][(c mod ncg) * 128 + col]; salient
// chunks take the column from the VCM index table staged in LDS (0xFFFF: padding column). xrow is the thread's byte
// offset of its batch row in x. Every load is unconditional and in bounds.
__device__ __forceinline__ void bat_stage_load(const GemmArgs& a, const uint16_t* s_xidx, const BatStageCursor& s,
                                               int n, uint32_t xrow, BatStage& r) {
  const int t = threadIdx.x;
  const int col = t & 255;
  const int half = col >> 7;
  const bool real = s.k < n;
  const int c = 2 * s.sc + half;
  uint32_t j;
  bool valid;
  if (c < a.ngc) {
    int cm = s.cm + half;
    if (cm == a.ncg) cm = 0;
    j = uint32_t(cm * 128 + (col & 127));
    valid = j < uint32_t(a.N);
  } else {
    const uint32_t idx = real ? uint32_t(s_xidx[s.k * 256 + col]) : 0xFFFFu;
    valid = idx != 0xFFFFu;
    j = idx;
  }
  valid = valid && real;
  j = valid ? j : 0u;
  const int cs_unit = real ? s.sc : 0;
  r.cs = *reinterpret_cast<const uint16_t*>(reinterpret_cast<const uint8_t*>(a.colscale) + cs_unit * 512 +
                                            uint32_t(col) * 2u);
  r.xb = *reinterpret_cast<const uint16_t*>(reinterpret_cast<const uint8_t*>(a.x) + xrow + j * 2u);
  r.ok = valid && (t >> 8) < a.B;
}

// Staged layout: chunk h of the unit, batch row b, column 8s + n at h*XC + (b*16 + s)*12 + n, so a build thread reads
// the 8 columns of its sub-vector with two 16-byte reads and the 16 sub-vectors of one batch row lie in 16 different
// groups of four LDS banks (the stride of 12 floats spreads them).
__device__ __forceinline__ void bat_stage_write(float* xs_slot, const BatStage& r) {
  const int t = threadIdx.x;
  const int b = t >> 8;
  const int col = t & 255;
  xs_slot[(col >> 7) * Bat::XC + (b * 16 + ((col & 127) >> 3)) * Bat::XSS + (col & 7)] =
      r.ok ? h2f(uint16_t(r.xb)) * h2f(uint16_t(r.cs)) : 0.f;
}

// Build the 16 tables (256 patterns x NB batch rows) of one staged chunk; entry (p, s, b) at (p*16 + s)*4 + b whatever
// NB is, so the lookups' addresses do not depend on it. NB = 4: thread t owns sub-vector s = t & 15, batch row
// b = (t >> 4) & 3 and the 16 patterns whose top four bits are t >> 6; NB = 2: b = (t >> 4) & 1 and the 8 patterns
// whose top five bits are t >> 5. Patterns are enumerated in Gray order (each entry is the previous one plus or minus
// 2*xv[n]).
template <int NB>
__device__ __forceinline__ void bat_build(float* tbl, const float* xs_chunk) {
  constexpr int LOW = NB == 4 ? 4 : 3;   // low pattern bits enumerated by one thread
  const int t = threadIdx.x;
  const int s = t & 15;
  const int b = (t >> 4) & (NB - 1);
  const int hi = t >> (NB == 4 ? 6 : 5);
  const float4 lo4 = *reinterpret_cast<const float4*>(xs_chunk + (b * 16 + s) * Bat::XSS);
  const float4 hi4 = *reinterpret_cast<const float4*>(xs_chunk + (b * 16 + s) * Bat::XSS + 4);
  const float xv[8] = {lo4.x, lo4.y, lo4.z, lo4.w, hi4.x, hi4.y, hi4.z, hi4.w};
  float v = 0.f;
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const bool plus = n >= LOW && ((hi >> (n - LOW)) & 1);
    v += plus ? xv[n] : -xv[n];
  }
  float d[LOW];
#pragma unroll
  for (int n = 0; n < LOW; ++n) d[n] = 2.f * xv[n];
  float* col = tbl + s * 4 + b;
  const int pbase = hi << LOW;
  col[pbase * 64] = v;
#pragma unroll
  for (int k = 1; k < (1 << LOW); ++k) {
    const int n = __builtin_ctz(k);
    const int gk = k ^ (k >> 1);
    v += ((gk >> n) & 1) ? d[n] : -d[n];
    col[(pbase | gk) * 64] = v;
  }
}

// Chunk J of the unit: the thread's sign words of that chunk are in stored slot J XOR [row mod 32 >= 16]; 16 lookups
// of NB batch values (one 16- or 8-byte LDS read each), times the chunk's row scale, into acc.
template <int J, int NB>
__device__ __forceinline__ void bat_lookup(const float* tbl, const BatRing& rg, const uint32_t (&cq)[4], bool swap,
                                           float (&acc)[1][NB]) {
  const uint32_t sh = (threadIdx.x & 1u) * 16u;
  const bool upper = (J == 1) != swap;
  float sum[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) sum[b] = 0.f;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const uint32_t w = upper ? rg.w[4 + m] : rg.w[m];
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
      const uint32_t addr = __builtin_amdgcn_perm(w, cq[m], sel);   // (p << 8) | (s << 4)
      if constexpr (NB == 4) {
        const float4 e = *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(tbl) + addr);
        sum[0] += e.x; sum[1] += e.y; sum[2] += e.z; sum[3] += e.w;
      } else {
        const float2 e = *reinterpret_cast<const float2*>(reinterpret_cast<const char*>(tbl) + addr);
        sum[0] += e.x; sum[1] += e.y;
      }
    }
  }
  const float rs = h2f(uint16_t(rg.r[J] >> sh));
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[0][b] = __builtin_fmaf(sum[b], rs, acc[0][b]);
}

template <int NB>
struct BatState {
  int n;                      // units of this workgroup
  int tile, sc;               // unit being looked up
  int first_tile, last_tile;
  bool first_shared, last_shared;
  int n_pending;
  float acc[1][NB];
};

// Row-scale plane of chunk 2*sc(k) + half of unit k (clamped to the MX staged units), from the table staged in LDS.
template <int MX>
__device__ __forceinline__ int32_t bat_plane(const int* s_planes, int k, int half) {
  return __builtin_amdgcn_readfirstlane(s_planes[2 * (k < MX ? k : MX - 1) + half]);
}

// Unit K of the workgroup (compile-time K, at most MX units: kBatMaxUnits, or kBigUnits for the instance of layers
// that would otherwise need a second wave of workgroups), in two sub-steps.
// Sub-step 0: request unit K+4's activations into a free set of staging registers and unit K+D's signs into the ring
// slot unit K-1 used (D+1 units of sign data in flight at every wait); build chunk 1's tables into buffer 1; look up
// chunk 0 (buffer 0).
// Sub-step 1: write unit K+2's activations (requested two units earlier) into the staging slot unit K no longer
// needs; build unit K+1's chunk 0 into buffer 0; look up chunk 1. Each wait covers loads that the step needs anyway:
// the staging loads waited for were issued before the sign loads of unit K+D-2.
template <int D, int K, int NB, int MX>
__device__ __forceinline__ void bat_units(const GemmArgs& a, BatState<NB>& st, BatCursor& cur, BatRing (&ring)[D + 1],
                                          BatStageCursor& scur, BatStage (&sr)[3], uint32_t xrow, float* tbl,
                                          float* xs, const uint16_t* s_xidx, const int* s_planes,
                                          const uint32_t (&cq)[4], bool swap) {
  if constexpr (K < MX) {
    if (K >= st.n) return;
    // sub-step 0
    bat_stage_load(a, s_xidx, scur, st.n, xrow, sr[(K + 4) % 3]);   // unit K+4
    bat_stage_cursor_next(a, scur);
    bat_issue_signs(a, cur, ring[(K + D) % (D + 1)]);
    bat_issue_rscale(a, cur, bat_plane<MX>(s_planes, K + D, 0), bat_plane<MX>(s_planes, K + D, 1),
                     ring[(K + D) % (D + 1)]);
    bat_cursor_advance(a, cur, K + D + 1 < st.n);
    bat_build<NB>(tbl + Bat::TBL, xs + (K & 1) * Bat::XS + Bat::XC);
    bat_lookup<0, NB>(tbl, ring[K % (D + 1)], cq, swap, st.acc);
    __syncthreads();
    // sub-step 1
    if (K + 2 < st.n) bat_stage_write(xs + (K & 1) * Bat::XS, sr[(K + 2) % 3]);
    if (K + 1 < st.n) bat_build<NB>(tbl, xs + ((K + 1) & 1) * Bat::XS);
    bat_lookup<1, NB>(tbl + Bat::TBL, ring[K % (D + 1)], cq, swap, st.acc);
    if (st.sc == a.steps - 1 || K + 1 == st.n) {
      const bool shared = st.tile == st.first_tile ? st.first_shared : (st.tile == st.last_tile && st.last_shared);
      if (shared) {
        store_partial<1024, 1, NB>(a, st.tile == st.first_tile ? 0 : 1, st.acc);
        ++st.n_pending;
      } else {
        store_tile_y<1024, 1, NB>(a, st.tile, st.acc);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) st.acc[0][b] = 0.f;
    }
    __syncthreads();
    if (++st.sc == a.steps) {
      st.sc = 0;
      ++st.tile;
    }
    bat_units<D, K + 1, NB, MX>(a, st, cur, ring, scur, sr, xrow, tbl, xs, s_xidx, s_planes, cq, swap);
  }
}

template <int D, int NB, bool R2, int MX = kBatMaxUnits>
__global__ void __launch_bounds__(1024) k_gemm_mu8_batch(GemmArgs args) {
  __shared__ __attribute__((aligned(16))) float tbl[2 * Bat::TBL];   // 128 KB: buffer 0 chunk 0, buffer 1 chunk 1
  __shared__ __attribute__((aligned(16))) float xs[2 * Bat::XS];      // staged activations, two units
  __shared__ uint16_t s_xidx[MX * 256];                                // VCM indices of the workgroup's units
  __shared__ int s_planes[2 * MX];                                     // row-scale planes of their chunks
  __shared__ int s_flag;

  // This workgroup's group of NB batch rows, with its own slice of the workspace (counters, then partial sums).
  GemmArgs a = args;
  const int grp = blockIdx.y;
  a.B = args.B - NB * grp < NB ? args.B - NB * grp : NB;
  a.x = args.x + int64_t(NB * grp) * args.ldx;
  a.y = static_cast<char*>(args.y) + int64_t(NB * grp) * args.ldy * (args.y_fp32 ? 4 : 2);
  a.counters = args.counters + int64_t(grp) * (((int64_t(args.n_tiles) * kCounterStride * 4 + 255) & ~255) / 4);
  a.partials = args.partials + int64_t(grp) * args.blocks * 2 * 1024 * NB;

  const int t = threadIdx.x;
  const int u0 = first_unit(a, blockIdx.x);
  const int u1 = first_unit(a, blockIdx.x + 1);
  BatState<NB> st;
  st.n = u1 - u0;
  st.tile = u0 / a.steps;
  st.sc = u0 - st.tile * a.steps;
  st.first_tile = st.tile;
  st.last_tile = (u1 - 1) / a.steps;
  st.first_shared = tile_is_shared(a, st.first_tile);
  st.last_shared = tile_is_shared(a, st.last_tile);
  st.n_pending = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) st.acc[0][b] = 0.f;
  const bool swap = ((t >> 4) & 1) != 0;   // rows with i mod 32 >= 16 hold the super-chunk's chunks swapped
  // byte offset of the thread's batch row in x (rows past B read row B-1; their values are masked)
  const uint32_t xrow = uint32_t(((t >> 8) < a.B ? (t >> 8) : a.B - 1) * a.ldx * 2);

  // VCM indices of the workgroup's units into LDS, if one of them has a salient chunk.
  bool has_sal = false;
  for (int k = 0, sc = st.sc; k < st.n; ++k) {
    has_sal |= 2 * sc + 1 >= a.ngc;
    if (++sc == a.steps) sc = 0;
  }
  if (has_sal) {
    constexpr int PER = MX * 256 / 1024;
    uint16_t xi[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int k = (t >> 8) + 4 * m;
      int sc = st.sc + k;
      while (sc >= a.steps) sc -= a.steps;
      xi[m] = a.xidx[sc * 256 + (t & 255)];
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) s_xidx[((t >> 8) + 4 * m) * 256 + (t & 255)] = xi[m];
    __syncthreads();
  }

  // Prologue order: the row-scale planes of the workgroup's chunks (lane 2k+h of a register loads unit k's chunk
  // 2sc+h; units past the range repeat valid chunks; the launch plan keeps n <= MX), the activations of
  // units 0 and 1, the sign data of units 0..D-1, then (each wait covering only older loads) their row scales once the
  // planes are in, the staging of units 0 and 1, and units 2 and 3's activations into the staging registers. The
  // planes reach LDS for the steps through the barrier before the first table build.
  int32_t planes;
  {
    const int lane = t & 63;
    int sc = st.sc + (lane >> 1) % MX;
    while (sc >= a.steps) sc -= a.steps;
    planes = a.chunk_plane[2 * sc + (lane & 1)];
  }
  BatStageCursor scur;
  scur.k = 0;
  scur.sc = st.sc;
  scur.cm = (2 * st.sc) % a.ncg;
  BatStage r0, r1;
  bat_stage_load(a, s_xidx, scur, st.n, xrow, r0);
  bat_stage_cursor_next(a, scur);
  bat_stage_load(a, s_xidx, scur, st.n, xrow, r1);
  bat_stage_cursor_next(a, scur);
  BatCursor cur;
  bat_cursor_init(a, cur, st.tile, st.sc);
  BatCursor cur0 = cur;
  BatRing ring[D + 1];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    bat_issue_signs(a, cur, ring[k]);
    bat_cursor_advance(a, cur, k + 1 < st.n);
  }
#pragma unroll
  for (int k = 0; k < D; ++k) {
    bat_issue_rscale(a, cur0, __builtin_amdgcn_readlane(planes, 2 * k), __builtin_amdgcn_readlane(planes, 2 * k + 1),
                     ring[k]);
    bat_cursor_advance(a, cur0, k + 1 < st.n);
  }
  if (t < 2 * MX) s_planes[t] = planes;
  bat_stage_write(xs, r0);
  bat_stage_write(xs + Bat::XS, r1);
  BatStage sr[3];
  bat_stage_load(a, s_xidx, scur, st.n, xrow, sr[2]);   // unit 2
  bat_stage_cursor_next(a, scur);
  bat_stage_load(a, s_xidx, scur, st.n, xrow, sr[0]);   // unit 3
  bat_stage_cursor_next(a, scur);
  // Per-lane byte offsets of the table columns read at step q: sub-vector (q + t) mod 16 (rows are t mod 16).
  uint32_t cq[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    cq[m] = 0u;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) cq[m] |= (((uint32_t(4 * m + bb) + uint32_t(t)) & 15u) << 4) << (8 * bb);
  }
  __syncthreads();
  bat_build<NB>(tbl, xs);   // unit 0, chunk 0
  __syncthreads();
  bat_units<D, 0, NB, MX>(a, st, cur, ring, scur, sr, xrow, tbl, xs, s_xidx, s_planes, cq, swap);
  if constexpr (!R2) {   // else the split tiles are reduced by k_reduce_split after this kernel
    const int pend0 = st.first_shared ? st.first_tile : st.last_tile;
    publish_pending<1024, 1, NB>(a, pend0, st.last_tile, st.n_pending, &s_flag);
  }
}

template <int NB>
static bool launch_batch_nb(const GemmArgs& a, int n_groups, int depth, bool reduce2, int mx, hipStream_t stream) {
  const dim3 grid(unsigned(a.blocks), unsigned(n_groups));
  if (mx == kBigUnits) {   // the launch plan takes it with the second-kernel reduction only
    if (!reduce2 || n_groups != 1 || depth != 1) return false;
    hipLaunchKernelGGL((k_gemm_mu8_batch<1, NB, true, kBigUnits>), grid, dim3(1024), 0, stream, a);
    launch_reduce_split(a, NB, 1024, stream);
    return true;
  }
  if (reduce2) {   // one batch group, depth 1 (launch plan): the partial sums are laid out as k_reduce_split reads them
    if (n_groups != 1 || depth != 1) return false;
    hipLaunchKernelGGL((k_gemm_mu8_batch<1, NB, true>), grid, dim3(1024), 0, stream, a);
    launch_reduce_split(a, NB, 1024, stream);
    return true;
  }
  switch (depth) {
    case 1: hipLaunchKernelGGL((k_gemm_mu8_batch<1, NB, false>), grid, dim3(1024), 0, stream, a); return true;
    case 2: hipLaunchKernelGGL((k_gemm_mu8_batch<2, NB, false>), grid, dim3(1024), 0, stream, a); return true;
    case 3: hipLaunchKernelGGL((k_gemm_mu8_batch<3, NB, false>), grid, dim3(1024), 0, stream, a); return true;
  }
  return false;
}

bool launch_gemm_batch(const GemmArgs& a, int n_groups, int depth, int nb, bool reduce2, int mx, hipStream_t stream) {
  if (n_groups < 1 || n_groups > 4) return false;
  if (nb == 2) return n_groups == 1 && launch_batch_nb<2>(a, n_groups, depth, reduce2, mx, stream);
  if (nb == 4) return launch_batch_nb<4>(a, n_groups, depth, reduce2, mx, stream);
  return false;
}

}  // namespace fluxbin
