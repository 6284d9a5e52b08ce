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

#include "fluxbin_device.h"

namespace fluxbin {

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
//
// Pipeline per workgroup: a register ring of D+1 units of sign words and row scales; unit k+D is requested while the
// tables of unit k+1 are built (other LDS buffer) and unit k is looked up, so D+1 units of sign data are in flight at
// every wait. The folded
// activations of all the workgroup's units (at most XV = b1_max_units(NT), guaranteed by the launch plan) are staged in LDS first.
// =====================================================================================================================


// XU: most units a workgroup stages (the launch plan keeps every workgroup within it): b1_max_units(NT), or
// kBigUnits for the 1024-thread instance of layers that would otherwise need a second wave of workgroups.
template <int NT, int RPT, int XU = b1_max_units(NT)>
struct B1 {
  static constexpr int R = NT * RPT;
  static constexpr int NHI = NT / 32;                                   // pattern ranges per (slot, s) in the build
  static constexpr int LO = NHI == 4 ? 6 : (NHI == 8 ? 5 : (NHI == 16 ? 4 : 3));
  static constexpr int E = 1 << LO;                                     // entries per thread per build
  static constexpr int XV = XU;                                         // units staged in LDS (1 KB each)
  static constexpr int KPT = XV / (NT / 256);                           // staged units per thread
};

template <int RPT, int FG = 0>
struct Ring {
  uint32_t w[RPT][8];   // sign words of the thread's rows: [0..3] first stored chunk, [4..7] second
  uint32_t ra[RPT];     // 32-bit word holding the fp16 row scales of rows (i & ~1, i | 1) for chunk 2sc
  uint32_t rb[RPT];     // same for chunk 2sc+1
  // layers with FG (8 or 16) fine salient row-scale groups per chunk: the FG fp16 scales of the thread's row for each
  // stored slot (slot h at f[j][h*FG/2 ..]), already in position-block order
  uint32_t f[FG ? RPT : 1][FG ? FG : 1];
};

// Super-chunk index sc0 + k of a workgroup's unit k, wrapped at the end of the tile: v < steps + XV, so one
// subtraction suffices unless the layer has fewer than XV super-chunks (then the remainder).
__device__ __forceinline__ int wrap_sc(int v, int steps) {
  if (v >= steps) v -= steps;
  if (v >= steps) v %= steps;
  return v;
}

// Stage the folded activations xv = x[j] * colscale of the n <= XV units starting at super-chunk sc0 into
// xs[k*256 + col] (super-chunks wrap around at the end of a tile). Global chunks read x[j] directly (j follows from the
// chunk index); salient chunks read their input column from the VCM index table first (Eq. 13), then gather it.
// stage_issue() issues the loads. stage_write_global() waits for them (nothing else is in flight yet, so this is one
// short round trip), writes the global and padding columns and issues the salient gathers; the sign loads follow, and
// stage_write_salient() writes the gathered columns of a range of units when they are needed (waiting for the gathers
// never waits for sign data, which was requested after them).
// Every wavefront covers 64 columns of one half (one chunk) of each of its units, so the unit, its super-chunk, the
// chunk and whether it is salient are wavefront-uniform (scalar) values; only the column within the chunk is per lane.
// All 16 wavefronts of a workgroup run this prologue at once, so it is kept free of divisions and loops: its scalar
// instructions, issued for every wavefront, delay the first sign requests of the last wavefronts.
template <int NT, int XU>
struct Staged {
  uint32_t v[B1<NT, 1, XU>::KPT];    // x bits (global column) or the index (salient column)
  uint32_t cs[B1<NT, 1, XU>::KPT];   // column scale bits
  uint32_t g[B1<NT, 1, XU>::KPT];    // gathered x bits of salient columns
  uint32_t sal;                  // bit m: the wavefront's chunk of its m-th staged unit is salient (or padding)
  uint32_t pad;                  // bit m: this lane's column of a global chunk is past the N input columns
  int32_t plane;                 // threads t < 2*XV: row-scale plane of chunk 2*sc(t/2) + (t&1)
};

// k-th staged unit of this thread's wavefront (wavefront-uniform).
template <int NT>
__device__ __forceinline__ int staged_unit(int m) {
  return (__builtin_amdgcn_readfirstlane(int(threadIdx.x)) >> 8) + m * (NT / 256);
}

template <int NT, int XU>
__device__ __forceinline__ void stage_issue(const GemmArgs& a, Staged<NT, XU>& sg, const int2* s_unit) {
  using P = B1<NT, 1, XU>;
  const int t = threadIdx.x;
  const int col = t & 255;
  const int half = (__builtin_amdgcn_readfirstlane(t) >> 7) & 1;   // chunk of the super-chunk this wavefront covers
  sg.sal = 0u;
  sg.pad = 0u;
#pragma unroll
  for (int m = 0; m < P::KPT; ++m) {   // unconditional, always in-bounds loads: all in flight at once
    const int k = staged_unit<NT>(m);
    const int2 u = s_unit[2 * k + half];
    const int jb = __builtin_amdgcn_readfirstlane(u.x);   // column base within the input, or -1: salient chunk
    const int c = __builtin_amdgcn_readfirstlane(u.y);    // chunk
    const int v = c * 128 + (col & 127);                   // virtual column
    const bool sal = jb < 0;
    const int j = jb + (col & 127);
    const bool pad = !sal && j >= a.N;
    // one unconditional load per unit (a select of addresses, not of loads, so that no load waits for another)
    sg.v[m] = uint32_t(*(sal ? a.xidx + v : a.x + (pad ? 0 : j)));
    sg.cs[m] = a.colscale[v];
    sg.sal |= uint32_t(sal) << m;
    sg.pad |= uint32_t(pad) << m;
  }
  sg.plane = 0;
  if (t < 2 * P::XV) sg.plane = a.chunk_plane[s_unit[t].y];
}

template <int NT, int XU>
__device__ __forceinline__ void stage_write_global(const GemmArgs& a, Staged<NT, XU>& sg, float* xs, int64_t* s_roff,
                                                   int sc0, int n) {
  using P = B1<NT, 1, XU>;
  const int t = threadIdx.x;
  const int col = t & 255;
  if (t < 2 * P::XV) s_roff[t] = int64_t(sg.plane) * a.Mp * 2;
#pragma unroll
  for (int m = 0; m < P::KPT; ++m) {
    const int k = staged_unit<NT>(m);
    const bool sal = (sg.sal >> m) & 1u;
    // unconditional, always in-bounds gather (x[0] for the other columns)
    sg.g[m] = a.x[(sal && sg.v[m] != 0xFFFFu) ? sg.v[m] : 0u];
    if (k < n && !sal) xs[k * 256 + col] = ((sg.pad >> m) & 1u) ? 0.f : h2f(uint16_t(sg.v[m])) * h2f(uint16_t(sg.cs[m]));
  }
}

template <int NT, int XU>
__device__ __forceinline__ void stage_write_salient(const GemmArgs& a, const Staged<NT, XU>& sg, float* xs, int sc0,
                                                    int n, int k_begin, int k_end) {
  using P = B1<NT, 1, XU>;
  const int t = threadIdx.x;
  const int col = t & 255;
#pragma unroll
  for (int m = 0; m < P::KPT; ++m) {
    const int k = staged_unit<NT>(m);
    if (k >= k_begin && k < k_end && k < n && ((sg.sal >> m) & 1u))
      xs[k * 256 + col] = sg.v[m] == 0xFFFFu ? 0.f : h2f(uint16_t(sg.g[m])) * h2f(uint16_t(sg.cs[m]));
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

// mu = 4: the 2 x 32 tables (16 entries each) of one super-chunk into buffer BUF. Layout (floats): buffer BUF at
// BUF*2048, chunk h at h*1024, entry (p, u) at p*64 + u and again at p*64 + u + 32, so that a lookup of sub-vector
// (base + j) mod 32 is the address p*64 + base + j with no wrap (j < 8 an immediate). Entry e of the 1024 is
// (h, p, u) = (e >> 9, (e >> 5) & 15, e & 31): the sum of the sub-vector's four folded activations with the signs of p.
template <int NT, int BUF>
__device__ __forceinline__ void build_b1_mu4(float* lut, const float* xv256) {
#pragma unroll
  for (int e0 = 0; e0 < 1024; e0 += NT) {
    const int e = e0 + int(threadIdx.x);
    const int h = e >> 9, p = (e >> 5) & 15, u = e & 31;
    const float4 x4 = *reinterpret_cast<const float4*>(xv256 + h * 128 + 4 * u);
    const float v = ((p & 1) ? x4.x : -x4.x) + ((p & 2) ? x4.y : -x4.y) + ((p & 4) ? x4.z : -x4.z) +
                    ((p & 8) ? x4.w : -x4.w);
    float* dst = lut + BUF * 2048 + h * 1024 + p * 64 + u;
    dst[0] = v;
    dst[32] = v;
  }
}

// Request cursor: the unit (tile, sc) to request next, the uniform base of its sign slots, and the per-thread byte
// offsets of the thread's rows in the sign and row-scale sections for that tile. Rows past the packed rows (only in
// the last tile) read the last packed row: their sums are never stored.
template <int NT, int RPT>
struct Cursor {
  int tile, sc;
  const uint8_t* sbase;     // signs + 2*sc*Mp*16
  uint32_t soff[RPT];       // row * 16
  uint32_t roff[RPT];       // (row >> 1) * 4
};

template <int NT, int RPT>
__device__ __forceinline__ void cursor_rows(const GemmArgs& a, Cursor<NT, RPT>& c) {
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int row_raw = c.tile * (NT * RPT) + int(threadIdx.x) + NT * j;
    const uint32_t row = uint32_t(row_raw < a.Mp ? row_raw : a.Mp - 1);
    c.soff[j] = row * 16u;
    c.roff[j] = (row >> 1) * 4u;
  }
}

template <int NT, int RPT>
__device__ __forceinline__ void cursor_init(const GemmArgs& a, Cursor<NT, RPT>& c, int tile, int sc) {
  c.tile = tile;
  c.sc = sc;
  c.sbase = a.signs + int64_t(2 * sc) * a.Mp * 16;
  cursor_rows<NT, RPT>(a, c);
}

// Past the workgroup's last unit the pipeline keeps requesting (so that the number of loads in flight, which the
// waits count, is the same on every path): those requests read a 1 KB region at the start of the sign section and
// the first row-scale word, which stay cached.
template <int NT, int RPT>
__device__ __forceinline__ void cursor_dummy(const GemmArgs& a, Cursor<NT, RPT>& c) {
  c.sbase = a.signs;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    c.soff[j] = (threadIdx.x & 63u) * 16u;
    c.roff[j] = 0u;
  }
}

// Advances the cursor to the next unit, or to the dummy region when that unit is past the workgroup's range.
template <int NT, int RPT>
__device__ __forceinline__ void cursor_advance(const GemmArgs& a, Cursor<NT, RPT>& c, bool has_next);

template <int NT, int RPT>
__device__ __forceinline__ void cursor_next(const GemmArgs& a, Cursor<NT, RPT>& c) {
  if (++c.sc == a.steps) {
    c.sc = 0;
    ++c.tile;
    c.sbase = a.signs;
    cursor_rows<NT, RPT>(a, c);
  } else {
    c.sbase += int64_t(2) * a.Mp * 16;
  }
}

template <int NT, int RPT>
__device__ __forceinline__ void cursor_advance(const GemmArgs& a, Cursor<NT, RPT>& c, bool has_next) {
  if (has_next)
    cursor_next<NT, RPT>(a, c);
  else
    cursor_dummy<NT, RPT>(a, c);
}

// Issue the loads of the cursor's unit: sign words of both stored chunks (issue_signs) and the row-scale words of both
// chunks for row-scale planes pa, pb (issue_rscale), with uniform bases and the per-thread row offsets. Nothing here
// waits for them.
template <int NT, int RPT, int FG>
__device__ __forceinline__ void issue_signs(const GemmArgs& a, const Cursor<NT, RPT>& c, Ring<RPT, FG>& rg) {
  const uint8_t* e0 = c.sbase;
  const uint8_t* e1 = c.sbase + int64_t(a.Mp) * 16;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const uint4 v0 = load_stream16(e0 + c.soff[j]);
    const uint4 v1 = load_stream16(e1 + c.soff[j]);
    rg.w[j][0] = v0.x; rg.w[j][1] = v0.y; rg.w[j][2] = v0.z; rg.w[j][3] = v0.w;
    rg.w[j][4] = v1.x; rg.w[j][5] = v1.y; rg.w[j][6] = v1.z; rg.w[j][7] = v1.w;
  }
}

template <int NT, int RPT, int FG>
__device__ __forceinline__ void issue_rscale(const GemmArgs& a, const Cursor<NT, RPT>& c, int64_t oa, int64_t ob,
                                             Ring<RPT, FG>& rg) {
  const uint8_t* ba = reinterpret_cast<const uint8_t*>(a.rscale) + oa;
  const uint8_t* bb = reinterpret_cast<const uint8_t*>(a.rscale) + ob;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    rg.ra[j] = *reinterpret_cast<const uint32_t*>(ba + c.roff[j]);
    rg.rb[j] = *reinterpret_cast<const uint32_t*>(bb + c.roff[j]);
  }
}

// Fine salient row-scale groups (FG = 8 or 16 scales per chunk and row): the row's FG scales of the chunk held in each
// stored slot (slot h holds chunk 2sc + (h XOR hb)), from the chunk's block of rows of FG consecutive fp16 values
// (row * 2FG bytes in; c.soff = row * 16): FG/8 16-byte loads per slot.
template <int NT, int RPT, int FG>
__device__ __forceinline__ void issue_rscale_fine(const GemmArgs& a, const Cursor<NT, RPT>& c, int64_t oa, int64_t ob,
                                                  bool hb, Ring<RPT, FG>& rg) {
  static_assert(FG == 8 || FG == 16, "fine instances: 8 or 16 groups per chunk");
  const uint8_t* rs = reinterpret_cast<const uint8_t*>(a.rscale);
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const uint32_t off = c.soff[j] * uint32_t(FG / 8);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint8_t* p = rs + ((h != 0) != hb ? ob : oa) + off;
      uint32_t* d = &rg.f[j][h * (FG / 2)];
#pragma unroll
      for (int k = 0; k < FG / 8; ++k) {
        const uint4 v = *reinterpret_cast<const uint4*>(p + 16 * k);
        d[4 * k] = v.x; d[4 * k + 1] = v.y; d[4 * k + 2] = v.z; d[4 * k + 3] = v.w;
      }
    }
  }
}

template <int BUF>
__device__ __forceinline__ float lds_at(const float* lut, uint32_t byte_addr) {
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(lut) + byte_addr + BUF * 128);
}

// Sum of 16 lookups as a balanced tree: the reads are all issued before the first add, and the adds wait for pairs of
// results instead of one result each.
__device__ __forceinline__ float tree16(float (&v)[16]) {
#pragma unroll
  for (int w = 1; w < 16; w *= 2)
#pragma unroll
    for (int i = 0; i < 16; i += 2 * w) v[i] += v[i + w];
  return v[0];
}

template <int NT, int RPT, int BUF, int FG>
__device__ __forceinline__ void lookup_b1(const float* lut, const Ring<RPT, FG>& rg, const uint32_t (&c1)[4],
                                          const uint32_t (&c2)[4], bool hb, float (&acc)[RPT][1]) {
  const uint32_t sh = (threadIdx.x & 1u) * 16u;   // the rows of a thread have the parity of threadIdx.x
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    float v1[16], v2[16];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
        v1[4 * m + bb] = lds_at<BUF>(lut, __builtin_amdgcn_perm(rg.w[j][m], c1[m], sel));
      }
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
        v2[4 * m + bb] = lds_at<BUF>(lut, __builtin_amdgcn_perm(rg.w[j][4 + m], c2[m], sel));
      }
    }
    const float s1 = tree16(v1);
    const float s2 = tree16(v2);
    // s1 belongs to chunk 2sc + hb, s2 to the other one
    const float sa = hb ? s2 : s1;
    const float sb = hb ? s1 : s2;
    acc[j][0] = __builtin_fmaf(sa, h2f(uint16_t(rg.ra[j] >> sh)), acc[j][0]);
    acc[j][0] = __builtin_fmaf(sb, h2f(uint16_t(rg.rb[j] >> sh)), acc[j][0]);
  }
}

// Batch-1 lookups of a unit whose chunks have FG fine row-scale groups: the same 2 x 16 lookups as lookup_b1 (c1, c2
// hold the rotation of FG groups), each multiplied by the scale of its position block (positions q with the same
// q / (16 / FG)), in four chains of four FMAs per stored slot; one slot at a time, so that only one slot's lookups are
// live.
template <int NT, int RPT, int BUF, int FG>
__device__ __forceinline__ void lookup_b1_fine(const float* lut, const Ring<RPT, FG>& rg, const uint32_t (&c1)[4],
                                               const uint32_t (&c2)[4], float (&acc)[RPT][1]) {
  constexpr int N = 16 / FG;   // positions per group
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    float part[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float v[16];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
          const uint32_t sel = 0x0c0c0000u | ((4u + bb) << 8) | uint32_t(bb);
          v[4 * m + bb] = lds_at<BUF>(lut, __builtin_amdgcn_perm(rg.w[j][4 * h + m], h ? c2[m] : c1[m], sel));
        }
      }
      const uint32_t* f = &rg.f[j][h * (FG / 2)];
      float c[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float sum = 0.f;
#pragma unroll
        for (int q = 4 * k; q < 4 * k + 4; ++q) {
          const int slot = q / N;
          sum = __builtin_fmaf(v[q], h2f(uint16_t(f[slot >> 1] >> (16 * (slot & 1)))), sum);
        }
        c[k] = sum;
      }
      part[h] = (c[0] + c[1]) + (c[2] + c[3]);
    }
    acc[j][0] += part[0] + part[1];
  }
}

// mu = 4: chunk h of the unit is in stored slot h; nibble q of its 16 bytes (word q/8, bits 4(q%8)..) is sub-vector
// (q + i) mod 32 of row i. bm[m] = ((8m + t) mod 32) * 4 is the lane's byte column for word m, and nibble j of the word
// adds 4j (an immediate offset). Eight lookups per word, summed as a tree.
template <int NT, int RPT, int BUF, int FG>
__device__ __forceinline__ void lookup_b1_mu4(const float* lut, const Ring<RPT, FG>& rg, const uint32_t (&bm)[4],
                                              float (&acc)[RPT][1]) {
  const uint32_t sh = (threadIdx.x & 1u) * 16u;
  const char* base = reinterpret_cast<const char*>(lut) + BUF * 8192;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    float sum[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float part[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const uint32_t w = rg.w[j][4 * h + m];
        float v[8];
#pragma unroll
        for (int n = 0; n < 8; ++n) {
          const uint32_t addr = (__builtin_amdgcn_ubfe(w, 4 * n, 4) << 8) | bm[m];
          v[n] = *reinterpret_cast<const float*>(base + h * 4096 + 4 * n + addr);
        }
        part[m] = ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
      }
      sum[h] = (part[0] + part[1]) + (part[2] + part[3]);
    }
    acc[j][0] = __builtin_fmaf(sum[0], h2f(uint16_t(rg.ra[j] >> sh)), acc[j][0]);
    acc[j][0] = __builtin_fmaf(sum[1], h2f(uint16_t(rg.rb[j] >> sh)), acc[j][0]);
  }
}

// Byte offsets in the row-scale section of the planes of chunks 2*sc(k) and 2*sc(k)+1 of the workgroup's unit k
// (clamped to its last unit), from the table the prologue staged in LDS (one broadcast read; no scalar load is waited
// for inside the pipeline).
__device__ __forceinline__ void roff_of(const int64_t* s_roff, int k, int n, int64_t& oa, int64_t& ob) {
  const int kk = k < n ? k : n - 1;
  const int4 v = *reinterpret_cast<const int4*>(s_roff + 2 * kk);
  oa = int64_t((uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(v.y))) << 32) |
               uint32_t(__builtin_amdgcn_readfirstlane(v.x)));
  ob = int64_t((uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(v.w))) << 32) |
               uint32_t(__builtin_amdgcn_readfirstlane(v.z)));
}

// Per-workgroup state of the batch-1 kernel.
template <int NT, int RPT>
struct B1State {
  int n;                       // units of this workgroup
  int tile, sc;                // of the unit being looked up
  int first_tile, last_tile;   // tiles touched by this workgroup
  bool first_shared, last_shared;   // whether other workgroups contribute to them
  int n_pending;               // shared tiles whose partial sums await publication (first, then last)
  float acc[RPT][1];
};

// Step K of the pipeline (K = unit index within the workgroup): request unit K+D into ring slot (K+D) % (D+1) (the
// slot of unit K-1, looked up in the previous step), build unit K+1 into LDS buffer (K+1) % 2, look up unit K (slot
// K % (D+1), buffer K % 2). The prologue requests units 0..D-1, so D+1 units are in flight at every wait. The steps
// are unrolled at compile time (a workgroup has at most XV units) so that the wait before each lookup covers
// exactly the loads of unit K.
// Per-lane LUT address constants of the lookups (see the kernel): c1/c2 for chunks whose positions follow the plain
// rotation (one row scale per chunk, or 16 per chunk); with fine salient row-scale groups also the rotation of their
// group count (fs).
template <int FG>
struct LaneConsts {
  uint32_t c1[4], c2[4];
  uint32_t fs1[FG == 8 ? 4 : 1], fs2[FG == 8 ? 4 : 1];   // FG = 16 rotates like one group (c1, c2)
};

// Bytes (hb << 6) | (s << 2) of the sub-vectors s at positions 4m .. 4m+3 of lane t's rows for a chunk with G scale
// groups (n = 16/G positions per group: the groups rotated by floor(t/n), the positions in a group by t).
__device__ __forceinline__ void rotation_consts(int t, int G, bool hb, uint32_t (&c1)[4], uint32_t (&c2)[4]) {
  const int n = 16 / G;
  const int ln = __builtin_ctz(uint32_t(n));
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    uint32_t b1 = 0u, b2 = 0u;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const int q = 4 * m + bb;
      const uint32_t sv = uint32_t(((((q >> ln) + (t >> ln)) & (G - 1)) << ln) | ((q + t) & (n - 1)));
      b1 |= ((sv << 2) | (hb ? 0x40u : 0u)) << (8 * bb);
      b2 |= ((sv << 2) | (hb ? 0u : 0x40u)) << (8 * bb);
    }
    c1[m] = b1;
    c2[m] = b2;
  }
}

// Scales per chunk (1 or the fine count) of super-chunk sc: the salient chunks' layout from chunk nfc on.
__device__ __forceinline__ int unit_G(const GemmArgs& a, int sc) { return 2 * sc >= a.nfc ? a.Gcs : a.Gcg; }

// Row-scale loads of the cursor's unit. The fine instances (global chunks with one scale per chunk, salient chunks with
// FG fine groups) issue the same number of loads per row for every unit: FG = 8: one 16-byte load per slot, or the two
// scale words of the global layout; FG = 16: two 16-byte loads per slot, or the two scale words plus two loads of a
// word that stays cached. With the same count on both paths the compiler's waits before each lookup cover exactly the
// loads of the unit looked up (different counts made it wait for the loads of the unit requested ahead too).
template <int NT, int RPT, int FG>
__device__ __forceinline__ void issue_rscale_any(const GemmArgs& a, const Cursor<NT, RPT>& c, int64_t oa, int64_t ob,
                                                 bool hb, Ring<RPT, FG>& rg) {
  if constexpr (FG > 0) {
    if (2 * c.sc >= a.nfc) {
      issue_rscale_fine<NT, RPT, FG>(a, c, oa, ob, hb, rg);
    } else {
      issue_rscale<NT, RPT, FG>(a, c, oa, ob, rg);
      if constexpr (FG == 16) {
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
          rg.f[j][0] = *reinterpret_cast<const uint32_t*>(a.rscale);
          rg.f[j][8] = *reinterpret_cast<const uint32_t*>(a.rscale + 2);
        }
      }
    }
  } else {
    issue_rscale<NT, RPT, FG>(a, c, oa, ob, rg);
  }
}

template <int MU, int NT, int RPT, int D, int K, int FG, int XU>
__device__ __forceinline__ void steps_b1(const GemmArgs& a, B1State<NT, RPT>& st, Cursor<NT, RPT>& cur,
                                         Ring<RPT, FG> (&ring)[D + 1], float* lut, float* xs,
                                         const LaneConsts<FG>& lc, bool hb, const int64_t* s_roff,
                                         const Staged<NT, XU>& sg, int sc0) {
  constexpr int XV = XU;
  if constexpr (K < XV) {
    if (K >= st.n) return;
    constexpr int BUF = K & 1;
    constexpr int KI = (K + D) < XV ? (K + D) : XV - 1;   // unit requested (clamped)
    issue_signs<NT, RPT, FG>(a, cur, ring[(K + D) % (D + 1)]);
    int64_t oa, ob;
    roff_of(s_roff, KI, st.n, oa, ob);
    issue_rscale_any<NT, RPT, FG>(a, cur, oa, ob, hb, ring[(K + D) % (D + 1)]);
    cursor_advance<NT, RPT>(a, cur, K + D + 1 < st.n);
    if (K + 1 < st.n) {
      if constexpr (MU == 8)
        build_b1<NT, BUF ^ 1>(lut, xs + (K + 1) * 256);
      else
        build_b1_mu4<NT, BUF ^ 1>(lut, xs + (K + 1) * 256);
    }
    if constexpr (K == 0) stage_write_salient<NT, XU>(a, sg, xs, sc0, st.n, 2, XV);   // built from step 1 on
    if constexpr (MU == 8 && FG > 0) {
      if (2 * st.sc >= a.nfc) {
        if constexpr (FG == 16)
          lookup_b1_fine<NT, RPT, BUF, FG>(lut, ring[K % (D + 1)], lc.c1, lc.c2, st.acc);
        else
          lookup_b1_fine<NT, RPT, BUF, FG>(lut, ring[K % (D + 1)], lc.fs1, lc.fs2, st.acc);
      } else {
        lookup_b1<NT, RPT, BUF, FG>(lut, ring[K % (D + 1)], lc.c1, lc.c2, hb, st.acc);
      }
    } else if constexpr (MU == 8) {
      lookup_b1<NT, RPT, BUF, FG>(lut, ring[K % (D + 1)], lc.c1, lc.c2, hb, st.acc);
    } else {
      lookup_b1_mu4<NT, RPT, BUF, FG>(lut, ring[K % (D + 1)], lc.c1, st.acc);
    }
    if (st.sc == a.steps - 1 || K + 1 == st.n) {
      const bool shared = st.tile == st.first_tile ? st.first_shared : (st.tile == st.last_tile ? st.last_shared : false);
      if (shared) {
        store_partial<NT, RPT, 1>(a, st.tile == st.first_tile ? 0 : 1, st.acc);
        ++st.n_pending;
      } else {
        store_tile_y<NT, RPT, 1>(a, st.tile, st.acc);
      }
#pragma unroll
      for (int j = 0; j < RPT; ++j) st.acc[j][0] = 0.f;
    }
    __syncthreads();
    if (++st.sc == a.steps) {
      st.sc = 0;
      ++st.tile;
    }
    steps_b1<MU, NT, RPT, D, K + 1, FG, XU>(a, st, cur, ring, lut, xs, lc, hb, s_roff, sg, sc0);
  }
}

// FG > 0: the instances for layers whose salient chunks have FG = 8 or 16 fine row-scale groups (s = 16 or 8 salient
// columns per group, their global chunks one scale per chunk); mu = 8 only. Such layers need at most 128 VGPRs for
// four waves per SIMD (one 1024- or two 512-thread workgroups per CU), which the second launch bound (minimum waves
// per SIMD) asks of the compiler.
template <int MU, int NT, int RPT, int D, bool EARLY, int FG, int XU = b1_max_units(NT)>
__global__ void __launch_bounds__(NT, FG ? 4 : 1) k_gemv_b1(GemmArgs a) {
  static_assert(FG == 0 || MU == 8, "fine row-scale groups: mu = 8 only (mu = 4 layers with them run the generic kernel)");
  // mu = 8: 64 KB, two buffers interleaved per pattern; mu = 4: two buffers of 8 KB
  __shared__ __attribute__((aligned(16))) float lut[MU == 8 ? 256 * 64 : 2 * 2048];
  constexpr int XV = XU;
  __shared__ __attribute__((aligned(16))) float xs[XV * 256];  // staged folded activations
  __shared__ __attribute__((aligned(16))) int64_t s_roff[2 * XV];   // row-scale plane byte offsets, staged units
  __shared__ int s_flag;

  __shared__ int s_hdr[4];                                  // tile, sc, last tile, sharing flags
  __shared__ __attribute__((aligned(8))) int2 s_unit[2 * XV];   // per staged chunk: column base, chunk index

  const int t = threadIdx.x;
  const int u0 = first_unit(a, blockIdx.x);
  const int u1 = first_unit(a, blockIdx.x + 1);

  // Values that are the same for the whole workgroup are computed once, by the first wavefront, and read back by all
  // (16 wavefronts computing them each would spend their scalar issue slots on it while the first ones wait).
  if (t < 64) {
    const int n = u1 - u0;
    const int tile = u0 / a.steps;
    const int sc = u0 - tile * a.steps;
    int last_tile = tile;   // the last unit's tile without a division: sc + n - 1 < steps + XV
    int r = sc + n - 1;
    if (r >= a.steps) {
      r -= a.steps;
      ++last_tile;
      if (r >= a.steps) last_tile += r / a.steps;
    }
    if (t < 2 * XV) {   // staged chunk t: unit t/2 (wrapped at the end of the tile), half t&1
      const int c = 2 * wrap_sc(sc + (t >> 1), a.steps) + (t & 1);
      int cm = c;             // global chunk: its column block within its base, c mod ncg (Kb <= 4)
      if (cm >= a.ncg) cm -= a.ncg;
      if (cm >= a.ncg) cm -= a.ncg;
      if (cm >= a.ncg) cm -= a.ncg;
      s_unit[t] = make_int2(c < a.ngc ? cm * 128 : -1, c);
    }
    if (t == 0) {
      // a tile is shared unless this workgroup covers all of it (its units are one contiguous range)
      const bool fs = u0 != tile * a.steps || u1 < (tile + 1) * a.steps;
      const bool ls = u1 != (last_tile + 1) * a.steps || u0 > last_tile * a.steps;
      s_hdr[0] = tile;
      s_hdr[1] = sc;
      s_hdr[2] = last_tile;
      s_hdr[3] = int(fs) | (int(ls) << 1);
    }
  }
  __syncthreads();

  B1State<NT, RPT> st;
  st.n = u1 - u0;
  st.tile = __builtin_amdgcn_readfirstlane(s_hdr[0]);
  st.sc = __builtin_amdgcn_readfirstlane(s_hdr[1]);
  st.first_tile = st.tile;
  st.last_tile = __builtin_amdgcn_readfirstlane(s_hdr[2]);
  const int sh_flags = __builtin_amdgcn_readfirstlane(s_hdr[3]);
  st.first_shared = (sh_flags & 1) != 0;
  st.last_shared = (sh_flags & 2) != 0;
  st.n_pending = 0;
#pragma unroll
  for (int j = 0; j < RPT; ++j) st.acc[j][0] = 0.f;

  // Prologue: the activation, column-scale and plane-table loads. Large layers (not EARLY) stage the activations
  // before requesting any sign data: with every CU starting its sign stream at once, activation loads queued with it
  // would return only after the first burst; so the global columns are staged after one short round trip, then the
  // salient gathers and the sign loads of units 0..D-1 are issued. Small layers (EARLY) request the sign data of units
  // 0..D-1 right after the activation loads, so the round trips overlap; the salient gathers follow them. The row
  // scales of units 0..D-1 are requested after the first barrier, from the plane offsets staged in LDS (a unit's row
  // scales are used last, after all its lookups), and the tables of unit 0 are built right after.
  const bool hb = ((t >> 4) & 1) != 0;
  Staged<NT, XU> sg;
  const int sc0 = st.sc;
  stage_issue<NT, XU>(a, sg, s_unit);
  Cursor<NT, RPT> cur;
  cursor_init<NT, RPT>(a, cur, st.tile, st.sc);
  Ring<RPT, FG> ring[D + 1];
  Cursor<NT, RPT> cur0 = cur;
  if constexpr (!EARLY) stage_write_global<NT, XU>(a, sg, xs, s_roff, sc0, st.n);   // n <= XV (launch plan)
#pragma unroll
  for (int k = 0; k < D; ++k) {   // units 0..D-1 (the dummy region past the end)
    issue_signs<NT, RPT, FG>(a, cur, ring[k]);
    cursor_advance<NT, RPT>(a, cur, k + 1 < st.n);
  }
  if constexpr (EARLY) stage_write_global<NT, XU>(a, sg, xs, s_roff, sc0, st.n);

  // Per-lane byte offsets of the table columns read at step q: rows are congruent to t modulo 32. Byte bb of c1[m] is
  // (hb << 6) | (s << 2) with s = (t + 4m + bb) mod 16 (the four bytes at once: no byte exceeds 18 before the mask).
  // (mu = 4: c1[m] is the lane's byte column of word m, ((8m + t) mod 32) * 4; c2 and hb are not used.)
  // Salient chunks with fine row-scale groups rotate the positions by groups (rotation_consts).
  LaneConsts<FG> lc;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    if constexpr (MU == 8) {
      const uint32_t sb = ((((uint32_t(t) + 4u * m) & 15u) * 0x01010101u + 0x03020100u) & 0x0F0F0F0Fu) << 2;
      lc.c1[m] = sb | (hb ? 0x40404040u : 0u);
      lc.c2[m] = sb | (hb ? 0u : 0x40404040u);
    } else {
      lc.c1[m] = ((uint32_t(t) + 8u * m) & 31u) * 4u;
      lc.c2[m] = 0u;
    }
  }
  if constexpr (FG == 8) rotation_consts(t, FG, hb, lc.fs1, lc.fs2);

  stage_write_salient<NT, XU>(a, sg, xs, sc0, st.n, 0, 2);
  __syncthreads();
  // the row scales of units 0..D-1, from the plane offsets just staged (they are used last in a unit's lookups)
#pragma unroll
  for (int k = 0; k < D; ++k) {
    int64_t oa, ob;
    roff_of(s_roff, k, st.n, oa, ob);
    issue_rscale_any<NT, RPT, FG>(a, cur0, oa, ob, hb, ring[k]);
    cursor_advance<NT, RPT>(a, cur0, k + 1 < st.n);
  }
  if constexpr (MU == 8)
    build_b1<NT, 0>(lut, xs);
  else
    build_b1_mu4<NT, 0>(lut, xs);
  __syncthreads();
  steps_b1<MU, NT, RPT, D, 0, FG, XU>(a, st, cur, ring, lut, xs, lc, hb, s_roff, sg, sc0);
  const int pend0 = st.first_shared ? st.first_tile : st.last_tile;
  publish_pending<NT, RPT, 1>(a, pend0, st.last_tile, st.n_pending, &s_flag);
}

// Split tiles reduced by a second kernel over the whole chip, after a kernel that stored every contributor's partial
// sums and left the tile counters alone (the matrix-core small-batch kernel): one 256-thread workgroup per (split
// tile, padded batch row, 256 rows), one thread per row and batch row. The contributors' partial sums are added in
// workgroup order from +0, the order (hence the bits) of the counter protocol's reducer. With several batch rows a
// tile's partial sums are tens to hundreds of KB, which the counter protocol's one reducing workgroup reads through a
// single CU in dependent rounds; here they are read by all CUs at once. (For batch 1 the gap between the two kernels
// costs more than the counter protocol's reduction: measured 1.3-1.5 us slower on 4096- to 11008-row layers.)
__global__ void __launch_bounds__(256) k_reduce_split(GemmArgs a, int bp, int R) {
  constexpr int CH = 16;
  const int q = R >> 8;   // 256-row parts of a tile
  const int per_tile = bp * q;
  const int tile = int(blockIdx.x) / per_tile;
  const int rem = int(blockIdx.x) - tile * per_tile;
  const int b = rem / q;
  if (b >= a.B || !tile_is_shared(a, tile)) return;   // unshared tiles were stored by their owner
  const int r = (rem - b * q) * 256 + int(threadIdx.x);
  const int b_first = owner_of(a, tile * a.steps);
  const int n_c = owner_of(a, (tile + 1) * a.steps - 1) - b_first + 1;
  const bool first_in_slot1 = first_unit(a, b_first) < tile * a.steps;   // its range starts in an earlier tile
  float sum = 0.f;
  for (int c0 = 0; c0 < n_c; c0 += CH) {
    float v[CH];
#pragma unroll
    for (int k = 0; k < CH; ++k) {
      const int c = c0 + k;
      const int slot = (b_first + c) * 2 + ((c == 0 && first_in_slot1) ? 1 : 0);
      v[k] = c < n_c ? a.partials[(int64_t(slot) * bp + b) * R + r] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < CH; ++k) sum += v[k];
  }
  const int64_t row = int64_t(tile) * R + r;
  if (row < a.M) store_y(a, b, row, sum);
}

void launch_reduce_split(const GemmArgs& a, int bp, int R, hipStream_t stream) {
  hipLaunchKernelGGL(k_reduce_split, dim3(unsigned(a.n_tiles * bp * (R >> 8))), dim3(256), 0, stream, a, bp, R);
}

// Stream probe: the batch-1 kernel's sign and row-scale requests (same plan, cursor, ring depth and per-unit barrier)
// without the table work; each unit's words are folded into a checksum so the loads are not removed.
template <int NT, int D, int XU = b1_max_units(NT)>
__global__ void __launch_bounds__(NT) k_stream_probe(GemmArgs a, uint32_t* sink) {
  const int u0 = first_unit(a, blockIdx.x);
  const int u1 = first_unit(a, blockIdx.x + 1);
  const int n = u1 - u0;
  const int tile = u0 / a.steps;
  const int sc = u0 - tile * a.steps;
  Cursor<NT, 1> cur;
  cursor_init<NT, 1>(a, cur, tile, sc);
  Ring<1> ring[D + 1];
  uint32_t acc = 0;
  int sck = sc;
#pragma unroll
  for (int k = 0; k < D; ++k) {
    issue_signs<NT, 1, 0>(a, cur, ring[k]);
    const int32_t p0 = load_uniform_i32(a.chunk_plane, 2 * sck);
    issue_rscale<NT, 1, 0>(a, cur, int64_t(p0) * a.Mp * 2, int64_t(load_uniform_i32(a.chunk_plane, 2 * sck + 1)) * a.Mp * 2,
                        ring[k]);
    cursor_advance<NT, 1>(a, cur, k + 1 < n);
    if (++sck == a.steps) sck = 0;
  }
#pragma unroll
  for (int k = 0; k < XU; ++k) {   // n <= XU (launch plan); unrolled so the ring stays in registers
    if (k < n) {
      Ring<1>& nx = ring[(k + D) % (D + 1)];
      issue_signs<NT, 1, 0>(a, cur, nx);
      issue_rscale<NT, 1, 0>(a, cur, int64_t(load_uniform_i32(a.chunk_plane, 2 * sck)) * a.Mp * 2,
                          int64_t(load_uniform_i32(a.chunk_plane, 2 * sck + 1)) * a.Mp * 2, nx);
      cursor_advance<NT, 1>(a, cur, k + D + 1 < n);
      if (++sck == a.steps) sck = 0;
      const Ring<1>& r = ring[k % (D + 1)];
#pragma unroll
      for (int m = 0; m < 8; ++m) acc ^= r.w[0][m];
      acc ^= r.ra[0] ^ r.rb[0];
      __syncthreads();
    }
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x & 255] = acc;   // practically never: keeps the loads live
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

// Stage the folded activations of n <= XU units starting at (c, g) into xs[k*XV + col*BG + b]. Thread t handles
// column t % 128 of every staged unit; all index/scale loads are issued before the activation gathers.
template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void stage_xv_gen(const GemmArgs& a, float* xs, int c, int g, int n) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  static_assert(NT % 128 == 0, "whole columns per thread group");
  constexpr int KPT = (P::XU * 128 + NT - 1) / NT;   // (unit, column) pairs per thread
  const int t = threadIdx.x;
  const int col = t % 128;
  uint16_t xi[KPT], cs[KPT];
  int cu[KPT], gu[KPT];
  // walk the units; thread t takes units k = t/128, t/128 + NT/128, ...
  int cc = c, gg = g;
#pragma unroll
  for (int k = 0; k < P::XU; ++k) {
    if ((k % (NT / 128)) == (t / 128) && k / (NT / 128) < KPT) {
      const int m = k / (NT / 128);
      cu[m] = cc;
      gu[m] = gg;
      xi[m] = a.xidx[cc * 128 + col];          // unconditional, always in-bounds: all loads in flight at once
      cs[m] = a.colscale[cc * 128 + col];
    }
    if (++gg == NG) {
      gg = 0;
      if (++cc == a.NCP) cc = 0;
    }
  }
  uint16_t xr[KPT][BG];
#pragma unroll
  for (int m = 0; m < KPT; ++m)
#pragma unroll
    for (int b = 0; b < BG; ++b) {
      const int bat = gu[m] * BG + b;
      xr[m][b] = a.x[int64_t(bat < a.B ? bat : 0) * a.ldx + (xi[m] == 0xFFFFu ? 0 : xi[m])];
    }
#pragma unroll
  for (int m = 0; m < KPT; ++m) {
    const int k = m * (NT / 128) + t / 128;
    if (k < n) {
#pragma unroll
      for (int b = 0; b < BG; ++b) {
        const int bat = gu[m] * BG + b;
        xs[k * P::XV + col * BG + b] = (xi[m] != 0xFFFFu && bat < a.B) ? h2f(xr[m][b]) * h2f(cs[m]) : 0.f;
      }
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

// Loads chunk c's sign entries of the thread's rows and their row scales: the scale itself for a chunk with one scale
// per row (rs), or, for fine row-scale groups, nothing yet (the lookups read the scale of each position from the
// chunk's block of G scales per row).
template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void load_unit_gen(const GemmArgs& a, int tile, int c, uint32_t (&w)[RPT][4],
                                              uint32_t (&rs)[RPT]) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  const int t = threadIdx.x;
  const int cu = __builtin_amdgcn_readfirstlane(c);
  const int tl = __builtin_amdgcn_readfirstlane(tile);
  const int32_t plane = load_uniform_i32(a.chunk_plane, cu);
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int row_raw = tl * P::R + t + NT * j;
    const int row = row_raw < a.Mp ? row_raw : a.Mp - 1;   // rows past the packed ones are never stored
    const int h = (MU == 8) ? ((cu & 1) ^ ((t & 31) >= 16 ? 1 : 0)) : (cu & 1);
    const uint4 v = load_stream16(a.signs + ((int64_t(cu >> 1) * 2 + h) * a.Mp + row) * 16);
    w[j][0] = v.x; w[j][1] = v.y; w[j][2] = v.z; w[j][3] = v.w;
    const int G = cu >= a.nfc ? a.Gcs : a.Gcg;
    rs[j] = G == 1 ? a.rscale[int64_t(plane) * a.Mp + row] : 0u;
  }
}

// Lookups of chunk c (sub-vector at position q of row i: groups of n = SPC/G positions rotated by floor(i/n), the
// positions in a group by i; G = 1 is the plain rotation (q + i) mod SPC). One row scale per chunk: the lookups are
// summed, then scaled; fine groups: each lookup times the scale of its position block, read from the chunk's block.
template <int MU, int BG, int NG, int NT, int RPT>
__device__ __forceinline__ void lookup_gen(const GemmArgs& a, const float* tbl, const uint32_t (&w)[RPT][4],
                                           const uint32_t (&rs)[RPT], int tile, int c, int g,
                                           float (&acc)[RPT][BG * NG]) {
  using P = Gen<MU, BG, NG, NT, RPT>;
  const uint32_t t = threadIdx.x;
  const int G = c >= a.nfc ? a.Gcs : a.Gcg;
  const int n = P::SPC / G;
  const int ln = __builtin_ctz(uint32_t(n));
  const int32_t plane = load_uniform_i32(a.chunk_plane, c);
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int row_raw = tile * P::R + int(t) + NT * j;
    const int row = row_raw < a.Mp ? row_raw : a.Mp - 1;
    const uint16_t* fine = a.rscale + (int64_t(plane) * a.Mp + int64_t(row) * G);
    float sum[BG];
#pragma unroll
    for (int b = 0; b < BG; ++b) sum[b] = 0.f;
#pragma unroll
    for (int q = 0; q < P::SPC; ++q) {
      const uint32_t p = (w[j][q / (32 / MU)] >> (MU * (q % (32 / MU)))) & uint32_t(P::NP - 1);
      const uint32_t sv = ((((uint32_t(q) >> ln) + (t >> ln)) & uint32_t(G - 1)) << ln) | ((uint32_t(q) + t) & uint32_t(n - 1));
      float f[BG];
      read_vec<BG>(tbl + (p * P::SPC + sv) * BG, f);
      if (G == 1) {
#pragma unroll
        for (int b = 0; b < BG; ++b) sum[b] += f[b];
      } else {
        const float sq = h2f(fine[q >> ln]);
#pragma unroll
        for (int b = 0; b < BG; ++b) sum[b] = __builtin_fmaf(f[b], sq, sum[b]);
      }
    }
    const float rsc = G == 1 ? h2f(uint16_t(rs[j])) : 1.f;
#pragma unroll
    for (int gg = 0; gg < NG; ++gg) {
#pragma unroll
      for (int b = 0; b < BG; ++b) {
        const float upd = __builtin_fmaf(sum[b], rsc, acc[j][gg * BG + b]);
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

  const int64_t u0 = first_unit(a, blockIdx.x);
  const int64_t u1 = first_unit(a, blockIdx.x + 1);
  const int64_t first_tile = u0 / a.steps;
  const int rem0 = int(u0 - first_tile * a.steps);

  float acc[RPT][P::BP];
#pragma unroll
  for (int j = 0; j < RPT; ++j)
#pragma unroll
    for (int b = 0; b < P::BP; ++b) acc[j][b] = 0.f;
  uint32_t w[RPT][4], wn[RPT][4];
  uint32_t rs[RPT], rsn[RPT];

  int n_left = int(u1 - u0);
  int tile = int(first_tile), c = rem0 / NG, g = rem0 % NG;
  int pending0 = 0, pending1 = 0, n_pending = 0;
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
    lookup_gen<MU, BG, NG, NT, RPT>(a, tbl + buf * P::TBL, w, rs, tile, c, g, acc);
    if ((c == a.NCP - 1 && g == NG - 1) || n_left == 1) {
      if (tile_end<NT, RPT, P::BP>(a, tile, first_tile, acc)) {
        if (n_pending == 0) pending0 = tile; else pending1 = tile;
        ++n_pending;
      }
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
  publish_pending<NT, RPT, P::BP>(a, pending0, pending1, n_pending, &s_flag);
}

// =====================================================================================================================
// Launch
// =====================================================================================================================

template <int MU, int NT, int RPT, bool EARLY>
static bool launch_b1_d(const GemmArgs& a, int depth, int fg, hipStream_t stream) {
  const dim3 grid(unsigned(a.blocks));
  if (fg) {   // fine salient row-scale groups: mu = 8, 512 or 1024 threads, one unit ahead (launch plan)
    if constexpr (MU == 8 && NT != 256) {
      if (depth != 1) return false;
      if (fg == 16) hipLaunchKernelGGL((k_gemv_b1<8, NT, RPT, 1, EARLY, 16>), grid, dim3(NT), 0, stream, a);
      else if (fg == 8) hipLaunchKernelGGL((k_gemv_b1<8, NT, RPT, 1, EARLY, 8>), grid, dim3(NT), 0, stream, a);
      else return false;
      return true;
    }
    return false;
  }
  if constexpr (MU == 8) {
    switch (depth) {
      case 2: hipLaunchKernelGGL((k_gemv_b1<8, NT, RPT, 2, EARLY, 0>), grid, dim3(NT), 0, stream, a); return true;
      case 3: hipLaunchKernelGGL((k_gemv_b1<8, NT, RPT, 3, EARLY, 0>), grid, dim3(NT), 0, stream, a); return true;
      default: break;
    }
  }
  hipLaunchKernelGGL((k_gemv_b1<MU, NT, RPT, 1, EARLY, 0>), grid, dim3(NT), 0, stream, a);   // mu = 4: depth 1 only
  return true;
}

template <int MU, int NT, int RPT>
static bool launch_b1(const GemmArgs& a, int depth, bool early, int fg, int xv, hipStream_t stream) {
  if (xv == kBigUnits) {   // the launch plan takes it for mu = 8, 1024 threads, one unit ahead, staged first only
    if constexpr (MU == 8 && NT == 1024 && RPT == 1) {
      if (depth != 1 || early || fg) return false;
      hipLaunchKernelGGL((k_gemv_b1<8, 1024, 1, 1, false, 0, kBigUnits>), dim3(unsigned(a.blocks)), dim3(1024), 0,
                         stream, a);
      return true;
    }
    return false;
  }
  return early ? launch_b1_d<MU, NT, RPT, true>(a, depth, fg, stream)
               : launch_b1_d<MU, NT, RPT, false>(a, depth, fg, stream);
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

// The plan's split of the units over the workgroups (first_unit): aligned to tiles, kpt per tile, or balanced.
static void set_split(const Plan& p, GemmArgs& a) {
  a.kpt = p.kpt;
  const int64_t steps = p.units / p.n_tiles;
  a.uq = int32_t(p.kpt > 0 ? steps / p.kpt : p.units / p.blocks);
  a.ur = int32_t(p.kpt > 0 ? steps % p.kpt : p.units % p.blocks);
}

fluxbin_status launch_stream_probe(const fluxbin_layer& L, const Plan& p, uint32_t* d_sink, hipStream_t stream) {
  GemmArgs a{};
  const uint8_t* base = static_cast<const uint8_t*>(L.d_base);
  a.signs = base + L.off_signs;
  a.rscale = reinterpret_cast<const uint16_t*>(base + L.off_rscale);
  a.chunk_plane = reinterpret_cast<const int32_t*>(base + L.off_chunk_plane);
  a.units = int32_t(p.units);
  a.blocks = int32_t(p.blocks);
  set_split(p, a);
  a.M = int32_t(L.shape.M);
  a.Mp = int32_t(L.Mp);
  a.NSC = int32_t(L.NSC);
  a.NCP = int32_t(2 * L.NSC);
  a.steps = int32_t(p.units / p.n_tiles);
  a.n_tiles = int32_t(p.n_tiles);
  const dim3 grid(unsigned(p.blocks));
  bool ok = true;
  switch (p.xv == kBigUnits ? -1 : p.nt * 10 + p.depth) {
    case -1: hipLaunchKernelGGL((k_stream_probe<1024, 1, kBigUnits>), grid, dim3(1024), 0, stream, a, d_sink); break;
    case 10241: hipLaunchKernelGGL((k_stream_probe<1024, 1>), grid, dim3(1024), 0, stream, a, d_sink); break;
    case 10242: hipLaunchKernelGGL((k_stream_probe<1024, 2>), grid, dim3(1024), 0, stream, a, d_sink); break;
    case 10243: hipLaunchKernelGGL((k_stream_probe<1024, 3>), grid, dim3(1024), 0, stream, a, d_sink); break;
    case 5121: hipLaunchKernelGGL((k_stream_probe<512, 1>), grid, dim3(512), 0, stream, a, d_sink); break;
    case 5122: hipLaunchKernelGGL((k_stream_probe<512, 2>), grid, dim3(512), 0, stream, a, d_sink); break;
    case 5123: hipLaunchKernelGGL((k_stream_probe<512, 3>), grid, dim3(512), 0, stream, a, d_sink); break;
    case 2561: hipLaunchKernelGGL((k_stream_probe<256, 1>), grid, dim3(256), 0, stream, a, d_sink); break;
    case 2562: hipLaunchKernelGGL((k_stream_probe<256, 2>), grid, dim3(256), 0, stream, a, d_sink); break;
    case 2563: hipLaunchKernelGGL((k_stream_probe<256, 3>), grid, dim3(256), 0, stream, a, d_sink); break;
    default: ok = false;
  }
  if (!ok) return fail(FLUXBIN_ERR_UNSUPPORTED, "no stream probe instance for this launch plan");
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the stream probe");
  return FLUXBIN_OK;
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
  a.img = (p.kernel == 3 || p.kernel == 5) ? reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(d_ws) + p.ws_image_off)
                                           : nullptr;
  a.ldx = ldx;
  a.ldy = ldy;
  a.units = int32_t(p.units);
  a.blocks = int32_t(p.blocks);
  set_split(p, a);
  a.N = int32_t(L.shape.N);
  a.ncg = int32_t(L.Npad / kChunk);
  a.ngc = int32_t(L.shape.Kb * (L.Npad / kChunk));
  a.M = int32_t(L.shape.M);
  a.Mp = int32_t(L.Mp);
  a.NSC = int32_t(L.NSC);
  a.NCP = int32_t(2 * L.NSC);
  a.steps = int32_t(p.units / p.n_tiles);
  a.B = B;
  a.y_fp32 = y_fp32;
  a.n_tiles = int32_t(p.n_tiles);
  bool ok = true;
  const Derived d = derive(L.shape);
  a.nfc = int32_t(d.nfc);
  a.Gcg = int32_t(d.Gcg);
  a.Gcs = int32_t(d.Gcs);
  const bool fine = d.Gcg > 1 || d.Gcs > 1;
  const int fg = fine ? (d.Gcg == 1 ? int(d.Gcs) : -1) : 0;   // batch-1 fine instances: salient groups only
  if (p.kernel == 0) {
    switch (p.nt) {   // one row per thread (the launch plan's only choice for this kernel)
      case 256: ok = L.shape.mu == 8 ? launch_b1<8, 256, 1>(a, p.depth, p.early, fg, p.xv, stream)
                                     : launch_b1<4, 256, 1>(a, p.depth, p.early, fg, p.xv, stream); break;
      case 512: ok = L.shape.mu == 8 ? launch_b1<8, 512, 1>(a, p.depth, p.early, fg, p.xv, stream)
                                     : launch_b1<4, 512, 1>(a, p.depth, p.early, fg, p.xv, stream); break;
      case 1024: ok = L.shape.mu == 8 ? launch_b1<8, 1024, 1>(a, p.depth, p.early, fg, p.xv, stream)
                                      : launch_b1<4, 1024, 1>(a, p.depth, p.early, fg, p.xv, stream); break;
      default: ok = false;
    }
  } else if (p.kernel == 2) {
    ok = !fine && launch_gemm_batch(a, p.n_groups, p.depth, p.bg, p.reduce2, p.xv, stream);
  } else if (p.kernel == 3) {
    ok = !fine && launch_gemm_mfma(a, p.bpad, int(L.shape.mu), p.depth, p.reduce2, stream);
  } else if (p.kernel == 5) {
    ok = !fine && launch_gemm_mfma_rows(a, p.bpad, int(L.shape.mu), p.nt / 64, p.rows / 16, stream);
  } else if (p.kernel == 4) {
    ok = fg >= 0 && launch_gemv_rows(a, int(L.shape.mu), p.nt / 64, p.depth, fg, p.rows / 16, stream);
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
