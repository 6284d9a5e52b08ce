// Internal declarations shared by the host code and the HIP kernels of libfluxbin.
#pragma once

#include <cstdint>
#include <cstddef>

#include "fluxbin.h"

namespace fluxbin {

constexpr int kChunk = 128;             // virtual columns per chunk (16 bytes of signs per row)
constexpr uint32_t kMagic = 0x42584C46u;  // "FLXB"
constexpr int kMaxBatch = 16;          // batch rows of one launch (a batch tile)
constexpr int kMaxBatchMfma = 32;      // batch rows of one matrix-core launch on layers with one row scale per chunk
constexpr int kMaxBatchCall = 8192;     // batch rows of one call: larger batches run as batch tiles
constexpr int kRwMaxN = 16384;          // row-complete batch-1 kernel: input columns staged in LDS
constexpr int kRwSteps = 16;            // row-complete batch-1 kernel: super-chunks per wavefront
// Units per workgroup of the batch-1 kernel (its LDS staging capacity): 16 for 1024-thread workgroups (one per CU),
// 12 for the smaller ones (two or more share a CU's LDS).
constexpr int b1_max_units(int nt) { return nt == 1024 ? 16 : 12; }
// The instances that stage up to 24 units per 1024-thread workgroup (batch-1 mu = 8 kernel, LUT batch kernel), for
// layers that then fit one wave of workgroups (with 16 or 12 units they would need a second wave). Separate instances:
// the batch-1 prologue then issues six staging loads per thread instead of four, which costs the layers that fit 16.
constexpr int kBigUnits = 24;
constexpr int kBatMaxUnits = 12;        // units per workgroup of the small-batch mu = 8 kernel (its LDS index table)
constexpr int kMfMaxUnits = 16;         // units per workgroup of the matrix-core small-batch kernel (unrolled steps)
// Matrix-core kernel with bp padded batch rows (4, 8, 16 or 32): dwords per (chunk, column group, K step) block of a
// unit's staged activation pairs (bp rows x 4 pairs, and 4 dwords of padding so that the 64 dwords one wavefront's
// gathering threads write land in 64 different banks), and dwords of a super-chunk's activation image (the 32 blocks
// and the 128 column-scale pairs, rounded up to whole 1 KB LDS-direct requests).
constexpr int mf_xstride(int bp) { return 4 * bp + 4; }
constexpr int mf_image_dwords(int bp) { return (32 * mf_xstride(bp) + 128 + 255) / 256 * 256; }
// Row-complete matrix-core kernel (small layers, B = 2..8): super-chunks per wavefront (units unrolled), and its
// dynamic LDS: column-scale pairs of every chunk (64 dwords each), then nblk activation blocks (16 per column block of
// (4 bp + 4) dwords).
// The staging image (column-scale pairs, then activation blocks) is copied in whole 1 KB requests, so the LDS holds
// the image rounded up to 256 dwords, and at least 64 dwords past its end.
constexpr int kMrSteps = 8;
constexpr int64_t mfma_rows_image_dwords(int64_t ncp, int64_t nblk, int bp) {
  return (ncp * 64 + nblk * 16 * (4 * bp + 4) + 255) / 256 * 256;
}
constexpr int64_t mfma_rows_lds_bytes(int64_t ncp, int64_t nblk, int bp) {
  return (ncp * 64 + nblk * 16 * (4 * bp + 4) + 64 > mfma_rows_image_dwords(ncp, nblk, bp)
              ? ncp * 64 + nblk * 16 * (4 * bp + 4) + 64
              : mfma_rows_image_dwords(ncp, nblk, bp)) * 4;
}
// Tile counters of the split-tile reduction sit kCounterStride 32-bit words (256 bytes) apart: every workgroup
// publishes at the end of a launch, and device-scope atomics on one memory line are serialized (densely packed
// counters cost the batch-1 GEMV on 8192 x 28672 layers 0.3-0.5 us).
#ifndef FLUXBIN_COUNTER_STRIDE
#define FLUXBIN_COUNTER_STRIDE 64
#endif
constexpr int kCounterStride = FLUXBIN_COUNTER_STRIDE;
// Static scratch of fluxbin_lut_gemv_noalloc: a fixed region of tile counters (room for every layer with at most
// kNoallocMaxM rows), then partial sums.
constexpr uint64_t kNoallocCounterBytes = 65536;
constexpr int64_t kNoallocMaxM = int64_t(kNoallocCounterBytes / (uint64_t(kCounterStride) * 4u) - 4) * 256;

struct Derived {
  int64_t Npad, ncg, Sv, ncs, NC, NSC, NCP, V, Mp, Gr, Gs, NRP;
  // Row scales per chunk and row: 1 (a "coarse" chunk: one scale plane, possibly shared by several chunks) or
  // 128 / g for a group size g below 128 (a "fine" chunk: its own block of Gc scales per row). Gcg for the global
  // chunks, Gcs for the salient ones.
  int64_t Gcg, Gcs;
  int64_t ngcp;   // chunks before the first salient chunk: Kb * ncg global chunks, plus one inert separator chunk
                  // when Kb * ncg is odd and Gcg != Gcs (so that no super-chunk mixes two scale layouts)
  int64_t nfc;    // first chunk that uses the salient chunks' scale layout (ngcp with a salient part, else NCP)
  int64_t Pg;     // row-scale planes of the global bases (the salient planes follow)
};

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline uint64_t round_up256(uint64_t v) { return (v + 255u) & ~uint64_t(255u); }

// Scales per chunk for a row-scale group of g columns over `extent` columns: fine (128 / g) when the group is shorter
// than both a chunk and the extent, else coarse (1).
inline int64_t chunk_scales(int64_t g, int64_t extent) { return (g < kChunk && g < extent) ? kChunk / g : 1; }

inline Derived derive(const fluxbin_shape& s) {
  Derived d{};
  d.Npad = ceil_div(s.N, kChunk) * kChunk;
  d.ncg = d.Npad / kChunk;
  const bool sal = s.S > 0 && s.Ks > 0;
  d.Sv = sal ? ceil_div(s.S, kChunk) * kChunk : 0;
  d.ncs = d.Sv / kChunk;
  d.Gcg = chunk_scales(s.g_r, s.N);
  d.Gcs = sal ? chunk_scales(s.g_s, s.S) : 1;
  d.ngcp = s.Kb * d.ncg + ((sal && d.Gcg != d.Gcs && (s.Kb * d.ncg) % 2 == 1) ? 1 : 0);
  d.NC = d.ngcp + s.Ks * d.ncs;
  d.NSC = ceil_div(d.NC, 2);
  d.NCP = 2 * d.NSC;
  d.nfc = sal ? d.ngcp : d.NCP;
  d.V = kChunk * d.NCP;
  d.Mp = ceil_div(s.M, 64) * 64;
  d.Gr = ceil_div(s.N, s.g_r);
  d.Gs = sal ? ceil_div(s.S, s.g_s) : 0;
  d.Pg = d.Gcg == 1 ? s.Kb * d.Gr : s.Kb * d.ncg * d.Gcg;
  d.NRP = d.Pg + (sal ? (d.Gcs == 1 ? s.Ks * d.Gs : s.Ks * d.ncs * d.Gcs) : 0);
  return d;
}

struct Offsets {
  uint64_t signs, rscale, colscale, xidx, chunk_plane, sal_idx, total;
};

inline Offsets offsets(const fluxbin_shape& s, const Derived& d) {
  Offsets o{};
  uint64_t off = FLUXBIN_HEADER_BYTES;
  o.signs = off;       off += round_up256(uint64_t(d.NSC) * 2u * uint64_t(d.Mp) * 16u);
  o.rscale = off;      off += round_up256(uint64_t(d.NRP) * uint64_t(d.Mp) * 2u);
  o.colscale = off;    off += round_up256(uint64_t(d.V) * 2u);
  o.xidx = off;        off += round_up256(uint64_t(d.V) * 2u);
  o.chunk_plane = off; off += round_up256(uint64_t(d.NCP) * 4u);
  o.sal_idx = off;     off += round_up256(uint64_t(s.S > 1 ? s.S : 1) * 2u);
  o.total = off;
  return o;
}

// The 256-byte header at the start of a packed buffer (little-endian, all fields naturally aligned).
struct Header {
  uint32_t magic;
  uint32_t version;
  fluxbin_shape shape;   // 56 bytes
  int64_t Npad, Sv, NC, NSC, Mp, Gr, Gs, NRP;
  uint64_t off_signs, off_rscale, off_colscale, off_xidx, off_chunk_plane, off_sal_idx, total;
  uint8_t pad[256 - 8 - sizeof(fluxbin_shape) - 8 * 8 - 7 * 8];
};
static_assert(sizeof(Header) == 256, "header must be 256 bytes");

// ---- error reporting (thread-local message) ----
fluxbin_status fail(fluxbin_status s, const char* fmt, ...);
void clear_error();  // every entry point starts with it: the message describes the last failed call only
fluxbin_status hip_fail(int hip_error, const char* what);

// ---- launch plan of the GEMV/GEMM kernels ----
struct Plan {
  int kernel;       // 0 = batch-1 super-chunk kernel (mu 8 or 4), 1 = generic (any mu, any batch), 2 = mu8 batch 2..16,
                    // 3 = matrix-core small batch (mu 8 or 4, batch 2..32), 4 = row-complete batch-1 (few rows),
                    // 5 = row-complete matrix-core small batch (few rows, batch 2..8)
  int nt;           // threads per block
  int rpt;          // rows per thread
  int rows;         // rows per tile (nt * rpt)
  int64_t n_tiles;  // ceil(M / rows)
  int64_t units;    // work units (tile x chunk step [x batch group])
  int64_t blocks;   // grid size
  int bg;           // batch rows per LUT group (generic and small-batch kernels)
  int n_groups;     // batch groups
  int bpad;         // bg * n_groups
  int depth;        // units of sign data requested ahead of the one looked up
  bool early;       // batch-1 kernel: request sign data before staging the activations (small layers)
  bool reduce2;     // matrix-core kernel: split tiles reduced by a second kernel over the whole chip
  uint64_t ws_counters_off, ws_partials_off, ws_bytes;
  uint64_t ws_image_off;   // matrix-core kernel: activation images after the partial sums (0 for other kernels)
  int kpt;                 // split-tile kernels: workgroups per tile with tile-aligned unit ranges (0: balanced split)
  int xv;                  // batch-1 and LUT batch kernels: kBigUnits for the instance staging that many units, else 0
};

// allow_rows = false: never the row-complete batch-1 kernel (the stream probe follows the split-tile kernel's plan)
fluxbin_status make_plan(const fluxbin_layer& L, int B, Plan* p, bool allow_rows = true);

// ---- launchers (fluxbin_pack.hip, fluxbin_gemv.hip) ----
fluxbin_status launch_pack(const fluxbin_layer& L, const fluxbin_weights& dev_w, const int32_t* d_sal_idx,
                           hipStream_t stream);
fluxbin_status launch_gemm(const fluxbin_layer& L, const Plan& p, int B, const uint16_t* d_x, int64_t ldx,
                           void* d_y, int64_t ldy, int y_fp32, void* d_ws, hipStream_t stream);
fluxbin_status launch_fill_zero(void* d, size_t bytes, hipStream_t stream);
fluxbin_status launch_stream_probe(const fluxbin_layer& L, const Plan& p, uint32_t* d_sink, hipStream_t stream);
fluxbin_status gemv_noalloc(const fluxbin_layer& L, const uint16_t* d_x, void* d_y, int y_fp32, hipStream_t stream);
fluxbin_status launch_debug_indices(const fluxbin_layer& L, uint8_t* d_p, hipStream_t stream);
fluxbin_status launch_unpack(const fluxbin_layer& L, uint32_t* d_signs, uint32_t* d_dense, hipStream_t stream);

int device_cu_count();  // CUs of the current device (cached per device), or -1 on a HIP error

}  // namespace fluxbin
