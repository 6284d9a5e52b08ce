// Small-batch (B = 2..16) LUT-GEMM of libfluxbin for gfx950, mu = 8.
//
// What is computed is the same as the batch-1 kernel (Sec. 3.2, Eqs. 11-15) for every batch row b < B:
//   y[b, i] = sum_c rscale[plane(c)][i] * sum_{s < 16} LUT_{b,c,s}[p(i, c, s)],
//   LUT_{b,c,s}[p] = sum_n xv[b, 128c + 8s + n] (2 bit_n(p) - 1),   xv = x[xidx] * colscale.
// Each sign word is read from HBM once and used for every batch row (the tables are what grows with B).
//
// Work decomposition. A tile is 1024 rows (one row per thread of a 1024-thread workgroup); a unit is one tile times
// one 128-column chunk. Units are numbered tile-major and split into equal contiguous ranges, one per workgroup, as in
// the batch-1 kernel, and split tiles are reduced by the same counter protocol (fluxbin_device.h).
//
// A workgroup handles one group of (up to) four batch rows, blockIdx.y; larger batches launch one row of workgroups
// per group. The groups read the same sign data at nearly the same time, so HBM streams it about once (the 256 MB
// last-level cache serves the repeats), while the table work, which grows with B and bounds this kernel, spreads over
// all CUs. LDS holds two table buffers of 256 patterns x 16 sub-vectors x 4 batch rows (64 KB each): entry (p, s, b)
// at (p*16 + s)*4 + b, so one ds_read_b128 returns the four batch values of a lookup. By the packed format a lane of
// row i reads sub-vector (q + i) mod 16 at byte q, so any 16 consecutive lanes read 16 different sub-vectors, i.e. all
// 64 LDS banks once: the lookups are conflict-free. Step k builds the tables of unit k+1 in the other buffer and looks
// up unit k. The folded activations of a unit (128 columns x 4 batch rows, fp32) are staged through a two-slot LDS
// ring: they are requested two units ahead into registers and written one unit ahead, so neither wait stalls the sign
// stream.
#include <hip/hip_runtime.h>

#include "fluxbin_device.h"

namespace fluxbin {

struct Bat {
  static constexpr int NT = 1024;
  static constexpr int BPN = 4;              // batch rows per workgroup
  static constexpr int TBL = 256 * 16 * 4;  // floats per table buffer (64 KB)
  static constexpr int XSS = 12;            // floats per (batch row, sub-vector) in the staging layout (8 + pad)
  static constexpr int XS = BPN * 16 * XSS;  // floats per staged unit
};

// Unit cursor: tile and chunk of the unit to request next, and the thread's byte offsets for that unit.
struct BatCursor {
  const uint8_t* sbase;  // signs + (c >> 1) * 2 * Mp * 16
  uint32_t soff;         // (h * Mp + row) * 16, h = stored slot of chunk c for this row (below 2^32 since M <= 2^27)
  uint32_t roff;         // (row >> 1) * 4
  int tile, c;
};

__device__ __forceinline__ void bat_cursor_set(const GemmArgs& a, BatCursor& cu, int tile, int c) {
  const int t = threadIdx.x;
  cu.tile = tile;
  cu.c = c;
  const int row_raw = tile * 1024 + t;
  const uint32_t row = uint32_t(row_raw < a.Mp ? row_raw : a.Mp - 1);   // rows past M are never stored
  const uint32_t h = uint32_t(c & 1) ^ uint32_t((t >> 4) & 1);           // slot swap of rows with i mod 32 >= 16
  cu.sbase = a.signs + int64_t((c >> 1) * 2) * a.Mp * 16;
  cu.soff = (h * uint32_t(a.Mp) + row) * 16u;
  cu.roff = (row >> 1) * 4u;
}

// Next unit, or a small cached region past the workgroup's range (the requests continue so that the number of loads
// in flight, which the waits count, is the same on every path).
__device__ __forceinline__ void bat_cursor_advance(const GemmArgs& a, BatCursor& cu, bool has_next) {
  if (has_next) {
    int c = cu.c + 1, tile = cu.tile;
    if (c == a.NCP) {
      c = 0;
      ++tile;
    }
    bat_cursor_set(a, cu, tile, c);
  } else {
    cu.sbase = a.signs;
    cu.soff = (threadIdx.x & 63u) * 16u;
    cu.roff = 0u;
  }
}

struct BatRing {
  uint32_t w[4];  // the row's 16-byte sign entry of the unit's chunk
  uint32_t r;     // 32-bit word with the fp16 row scales of rows (i & ~1, i | 1) in the chunk's plane
};

__device__ __forceinline__ void bat_issue(const GemmArgs& a, const BatCursor& cu, int32_t plane, BatRing& rg) {
  const uint4 v = load_stream16(cu.sbase + cu.soff);
  rg.w[0] = v.x; rg.w[1] = v.y; rg.w[2] = v.z; rg.w[3] = v.w;
  const uint8_t* rb = reinterpret_cast<const uint8_t*>(a.rscale) + int64_t(plane) * a.Mp * 2;
  rg.r = *reinterpret_cast<const uint32_t*>(rb + cu.roff);
}

// Staging registers of one unit: thread t holds column t & 127 of batch row t >> 7 (rows 4..7 of the mapping idle).
struct BatStage {
  uint32_t xb;   // x bits
  uint32_t cs;   // column scale bits
  bool ok;       // a real activation (else the staged value is 0)
};

// Request the activations of unit (chunk c, index k in the workgroup). Global chunks read x[b][j] with j following
// from the chunk; salient chunks take j from the VCM index table staged in LDS (0xFFFF: padding column). Every load is
// unconditional and in bounds.
__device__ __forceinline__ void bat_stage_load(const GemmArgs& a, const uint16_t* s_xidx, int k, int c, bool real,
                                               BatStage& r) {
  const int t = threadIdx.x;
  const int col = t & 127;
  const int b = t >> 7;
  int j = 0;
  bool valid = false;
  if (real) {
    if (c < a.ngc) {
      j = (c - (c / a.ncg) * a.ncg) * 128 + col;
      valid = j < a.N;
    } else {
      const uint32_t idx = s_xidx[k * 128 + col];
      valid = idx != 0xFFFFu;
      j = valid ? int(idx) : 0;
    }
  }
  if (!valid) j = 0;
  r.cs = real ? a.colscale[c * 128 + col] : a.colscale[0];
  const int bl = b < a.B ? b : a.B - 1;
  r.xb = a.x[int64_t(bl) * a.ldx + j];
  r.ok = valid && b < a.B;
}

// Staged layout: batch row b, column 8s + n at (b*16 + s)*12 + n, so a build thread reads the 8 columns of its
// sub-vector with two 16-byte reads and the 16 sub-vectors of one batch row lie in 16 different groups of four LDS
// banks (the stride of 12 floats spreads them).
__device__ __forceinline__ void bat_stage_write(float* xs_slot, const BatStage& r) {
  const int t = threadIdx.x;
  const int b = t >> 7;
  const int col = t & 127;
  if (b < Bat::BPN)
    xs_slot[(b * 16 + (col >> 3)) * Bat::XSS + (col & 7)] = r.ok ? h2f(uint16_t(r.xb)) * h2f(uint16_t(r.cs)) : 0.f;
}

// Build the 16 tables (256 patterns x 4 batch rows) of a staged unit. Thread t owns sub-vector s = t & 15, batch row
// b = (t >> 4) & 3 and the 16 patterns whose top four bits are t >> 6, enumerated in Gray order (each entry is the
// previous one plus or minus 2*xv[n]). A wavefront writes 64 consecutive floats per entry step.
__device__ __forceinline__ void bat_build(float* tbl, const float* xs_slot) {
  const int t = threadIdx.x;
  const int s = t & 15;
  const int b = (t >> 4) & 3;
  const int hi = t >> 6;
  const float4 lo4 = *reinterpret_cast<const float4*>(xs_slot + (b * 16 + s) * Bat::XSS);
  const float4 hi4 = *reinterpret_cast<const float4*>(xs_slot + (b * 16 + s) * Bat::XSS + 4);
  const float xv[8] = {lo4.x, lo4.y, lo4.z, lo4.w, hi4.x, hi4.y, hi4.z, hi4.w};
  float v = 0.f;
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const bool plus = n >= 4 && ((hi >> (n - 4)) & 1);
    v += plus ? xv[n] : -xv[n];
  }
  float d[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) d[n] = 2.f * xv[n];
  float* col = tbl + s * 4 + b;
  const int pbase = hi << 4;
  col[pbase * 64] = v;
#pragma unroll
  for (int k = 1; k < 16; ++k) {
    const int n = __builtin_ctz(k);
    const int gk = k ^ (k >> 1);
    v += ((gk >> n) & 1) ? d[n] : -d[n];
    col[(pbase | gk) * 64] = v;
  }
}

// 16 lookups of four batch values, times the row scale, into acc.
__device__ __forceinline__ void bat_lookup(const float* tbl, const BatRing& rg, const uint32_t (&cq)[4],
                                           float (&acc)[1][Bat::BPN]) {
  const uint32_t sh = (threadIdx.x & 1u) * 16u;
  float4 s4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int m = 0; m < 4; ++m) {
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
      const uint32_t addr = __builtin_amdgcn_perm(rg.w[m], cq[m], sel);   // (p << 8) | (s << 4)
      const float4 e = *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(tbl) + addr);
      s4.x += e.x; s4.y += e.y; s4.z += e.z; s4.w += e.w;
    }
  }
  const float rs = h2f(uint16_t(rg.r >> sh));
  acc[0][0] = __builtin_fmaf(s4.x, rs, acc[0][0]);
  acc[0][1] = __builtin_fmaf(s4.y, rs, acc[0][1]);
  acc[0][2] = __builtin_fmaf(s4.z, rs, acc[0][2]);
  acc[0][3] = __builtin_fmaf(s4.w, rs, acc[0][3]);
}

struct BatState {
  int n;                      // units of this workgroup
  int tile, c;                // unit being looked up
  int first_tile;
  int pending0, pending1, n_pending;
  float acc[1][Bat::BPN];
};

__device__ __forceinline__ int bat_plane(const int* s_planes, int k, int n) {
  const int kk = k < n ? k : n - 1;
  return __builtin_amdgcn_readfirstlane(s_planes[kk]);
}

// Step K of the workgroup (compile-time K, at most kBatMaxUnits units): request unit K+1 into the ring slot unit K-1
// used, build unit K+1's tables in the other buffer, look up unit K, then write unit K+2's activations (requested
// during step K-1) into the staging slot unit K no longer needs and request unit K+3's.
template <int K>
__device__ __forceinline__ void bat_steps(const GemmArgs& a, BatState& st, BatCursor& cur, BatRing (&ring)[2],
                                          BatStage& sr, float* tbl, float* xs, const uint16_t* s_xidx,
                                          const int* s_planes, const uint32_t (&cq)[4]) {
  if constexpr (K < kBatMaxUnits) {
    if (K >= st.n) return;
    bat_issue(a, cur, bat_plane(s_planes, K + 1, st.n), ring[(K + 1) & 1]);
    bat_cursor_advance(a, cur, K + 2 < st.n);
    if (K + 1 < st.n) bat_build(tbl + ((K + 1) & 1) * Bat::TBL, xs + ((K + 1) & 1) * Bat::XS);
    bat_lookup(tbl + (K & 1) * Bat::TBL, ring[K & 1], cq, st.acc);
    if (K + 2 < st.n) bat_stage_write(xs + (K & 1) * Bat::XS, sr);
    int c3 = st.c + 3;
    while (c3 >= a.NCP) c3 -= a.NCP;
    bat_stage_load(a, s_xidx, K + 3, c3, K + 3 < st.n, sr);
    if (st.c == a.NCP - 1 || K + 1 == st.n) {
      if (tile_end<1024, 1, Bat::BPN>(a, st.tile, st.first_tile, st.acc)) {
        if (st.n_pending == 0) st.pending0 = st.tile; else st.pending1 = st.tile;
        ++st.n_pending;
      }
#pragma unroll
      for (int b = 0; b < Bat::BPN; ++b) st.acc[0][b] = 0.f;
    }
    __syncthreads();
    if (++st.c == a.NCP) {
      st.c = 0;
      ++st.tile;
    }
    bat_steps<K + 1>(a, st, cur, ring, sr, tbl, xs, s_xidx, s_planes, cq);
  }
}

__global__ void __launch_bounds__(1024) k_gemm_mu8_batch(GemmArgs args) {
  __shared__ __attribute__((aligned(16))) float tbl[2 * Bat::TBL];   // 128 KB
  __shared__ __attribute__((aligned(16))) float xs[2 * Bat::XS];      // staged activations, two units
  __shared__ uint16_t s_xidx[kBatMaxUnits * 128];                      // VCM indices of the workgroup's units
  __shared__ int s_planes[kBatMaxUnits];
  __shared__ int s_flag;

  // This workgroup's group of batch rows, with its own slice of the workspace (counters, then partial sums).
  GemmArgs a = args;
  const int grp = blockIdx.y;
  a.B = args.B - 4 * grp < 4 ? args.B - 4 * grp : 4;
  a.x = args.x + int64_t(4 * grp) * args.ldx;
  a.y = static_cast<char*>(args.y) + int64_t(4 * grp) * args.ldy * (args.y_fp32 ? 4 : 2);
  a.counters = args.counters + int64_t(grp) * (((args.n_tiles * 4 + 255) & ~255) / 4);
  a.partials = args.partials + int64_t(grp) * args.blocks * 2 * 1024 * Bat::BPN;

  const int t = threadIdx.x;
  const int u0 = first_unit(a, blockIdx.x);
  const int u1 = first_unit(a, blockIdx.x + 1);
  BatState st;
  st.n = u1 - u0;
  st.tile = u0 / a.NCP;
  st.c = u0 - st.tile * a.NCP;
  st.first_tile = st.tile;
  st.pending0 = st.pending1 = st.n_pending = 0;
#pragma unroll
  for (int b = 0; b < Bat::BPN; ++b) st.acc[0][b] = 0.f;

  // Row-scale planes and VCM indices of the workgroup's units (the launch plan keeps n <= kBatMaxUnits).
  if (t < kBatMaxUnits) {
    int c = st.c + t;
    while (c >= a.NCP) c -= a.NCP;
    s_planes[t] = a.chunk_plane[c];
  }
  bool has_sal = false;
  for (int k = 0, c = st.c; k < st.n; ++k) {
    has_sal |= c >= a.ngc;
    if (++c == a.NCP) c = 0;
  }
  if (has_sal) {
    constexpr int PER = kBatMaxUnits * 128 / 1024;
    uint16_t xi[PER];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int k = (t >> 7) + 8 * m;
      int c = st.c + k;
      while (c >= a.NCP) c -= a.NCP;
      xi[m] = a.xidx[c * 128 + (t & 127)];
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) s_xidx[((t >> 7) + 8 * m) * 128 + (t & 127)] = xi[m];
  }
  __syncthreads();

  // Sign data of unit 0, then the activations of units 0 and 1 (their wait follows the sign request, which unit 0
  // needs right after anyway), then unit 2's activations into the staging registers.
  BatCursor cur;
  bat_cursor_set(a, cur, st.tile, st.c);
  BatRing ring[2];
  bat_issue(a, cur, bat_plane(s_planes, 0, st.n), ring[0]);
  bat_cursor_advance(a, cur, 1 < st.n);
  {
    BatStage r0, r1;
    int c1 = st.c + 1;
    if (c1 == a.NCP) c1 = 0;
    bat_stage_load(a, s_xidx, 0, st.c, true, r0);
    bat_stage_load(a, s_xidx, 1, c1, 1 < st.n, r1);
    bat_stage_write(xs, r0);
    bat_stage_write(xs + Bat::XS, r1);
  }
  BatStage sr;
  {
    int c2 = st.c + 2;
    while (c2 >= a.NCP) c2 -= a.NCP;
    bat_stage_load(a, s_xidx, 2, c2, 2 < st.n, sr);
  }
  // Per-lane byte offsets of the table columns read at step q: sub-vector (q + t) mod 16 (rows are t mod 16).
  uint32_t cq[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    cq[m] = 0u;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) cq[m] |= (((uint32_t(4 * m + bb) + uint32_t(t)) & 15u) << 4) << (8 * bb);
  }
  __syncthreads();
  bat_build(tbl, xs);
  __syncthreads();
  bat_steps<0>(a, st, cur, ring, sr, tbl, xs, s_xidx, s_planes, cq);
  publish_pending<1024, 1, Bat::BPN>(a, st.pending0, st.pending1, st.n_pending, &s_flag);
}

bool launch_gemm_batch(const GemmArgs& a, int n_groups, hipStream_t stream) {
  if (n_groups < 1 || n_groups > 4) return false;
  hipLaunchKernelGGL(k_gemm_mu8_batch, dim3(unsigned(a.blocks), unsigned(n_groups)), dim3(1024), 0, stream, a);
  return true;
}

}  // namespace fluxbin
