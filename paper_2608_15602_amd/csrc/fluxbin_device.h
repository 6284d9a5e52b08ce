// Device-side pieces shared by the LUT-GEMV/GEMM kernels of libfluxbin: kernel arguments, the balanced split of
// the work units over workgroups, and the deterministic split-tile reduction (tile counters + partial sums).
#pragma once

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
  uint32_t* img;     // matrix-core kernel: per-call activation images of every super-chunk (workspace)
  int64_t ldx, ldy;
  int32_t units, blocks;
  int32_t uq, ur;    // units per workgroup: uq + 1 for the first ur workgroups, uq for the others
  int32_t M, Mp, NSC, NCP;
  int32_t steps;     // units per tile
  int32_t B;         // batch rows actually present
  int32_t y_fp32;
  int32_t n_tiles;
  int32_t N;         // input columns
  int32_t ncg;       // chunks per global base
  int32_t ngc;       // global chunks (Kb * ncg); chunks >= ngc are salient or padding
  int32_t nfc;       // first chunk with the salient chunks' row-scale layout
  int32_t Gcg, Gcs;  // row scales per chunk and row: global / salient layout (1, or 2..32 for fine groups)
  int32_t kpt;       // kpt > 0: workgroup b covers part b mod kpt of tile b / kpt (tile-aligned ranges); 0: the
                     // balanced split of all units (first_unit)
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float h2f(uint16_t u) { return static_cast<float>(__builtin_bit_cast(_Float16, u)); }

__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f)); }

__device__ __forceinline__ uint4 load_stream16(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Split of the units over the workgroups: workgroup b owns [first_unit(b), first_unit(b + 1)).
// kpt == 0: balanced over all units, uq + 1 units for b < ur and uq otherwise (uq >= 1).
// kpt > 0: aligned to tiles, workgroup b owns part j = b mod kpt of tile b / kpt, the steps units of a tile split as
// uq + 1 units for j < ur and uq otherwise (uq = steps / kpt >= 1, ur = steps mod kpt).
__device__ __forceinline__ int first_unit(const GemmArgs& a, int b) {
  int t = 0;
  if (a.kpt > 0) {
    t = b / a.kpt;
    b -= t * a.kpt;
  }
  return t * a.steps + b * a.uq + (b < a.ur ? b : a.ur);
}

__device__ __forceinline__ int owner_of(const GemmArgs& a, int u) {
  int t = 0;
  if (a.kpt > 0) {
    t = u / a.steps;
    u -= t * a.steps;
  }
  const int big = a.ur * (a.uq + 1);
  return t * a.kpt + (u < big ? u / (a.uq + 1) : a.ur + (u - big) / a.uq);
}

__device__ __forceinline__ void store_y(const GemmArgs& a, int b, int64_t row, float v) {
  if (a.y_fp32)
    static_cast<float*>(a.y)[b * a.ldy + row] = v;
  else
    static_cast<uint16_t*>(a.y)[b * a.ldy + row] = f2h(v);
}

// ---------------------------------------------------------------------------------------------------------------------
// End of a tile's contribution from one workgroup.
//
// tile_end() (store_tile_y / store_partial): if the workgroup covers the whole tile it stores y directly; otherwise it stores its partial sums with
// device-coherent (agent-scope) stores into its slot (0 for its first tile, 1 for its last one) and returns true:
// the tile is then "pending". Nothing waits here, so the prefetched sign loads stay in flight.
// publish_pending(): once the workgroup has waited for all its memory operations, thread 0 bumps the counters of its
// pending tiles; the workgroup that brings a counter to the number of contributors adds the partial sums of all
// contributors in workgroup order (a fixed order, so y is the same on every run), stores y and resets the counter.
// ---------------------------------------------------------------------------------------------------------------------

// Whether workgroups other than the tile's first owner contribute to tile T.
__device__ __forceinline__ bool tile_is_shared(const GemmArgs& a, int tile) {
  return owner_of(a, tile * a.steps) != owner_of(a, (tile + 1) * a.steps - 1);
}

template <int NT, int RPT, int BP>
__device__ __forceinline__ void store_tile_y(const GemmArgs& a, int64_t tile, const float (&acc)[RPT][BP]) {
  const int64_t R = int64_t(NT) * RPT;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int64_t row = tile * R + threadIdx.x + NT * j;
    if (row < a.M) {
#pragma unroll
      for (int b = 0; b < BP; ++b)
        if (b < a.B) store_y(a, b, row, acc[j][b]);
    }
  }
}

template <int NT, int RPT, int BP>
__device__ __forceinline__ void store_partial(const GemmArgs& a, int slot, const float (&acc)[RPT][BP]) {
  const int64_t R = int64_t(NT) * RPT;
  float* mine = a.partials + ((int64_t(blockIdx.x) * 2 + slot) * BP) * R;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
#pragma unroll
    for (int b = 0; b < BP; ++b)
      __hip_atomic_store(mine + b * R + threadIdx.x + NT * j, acc[j][b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int NT, int RPT, int BP>
__device__ __forceinline__ bool tile_end(const GemmArgs& a, int64_t tile, int64_t first_tile, const float (&acc)[RPT][BP]) {
  if (!tile_is_shared(a, int(tile))) {
    store_tile_y<NT, RPT, BP>(a, tile, acc);
    return false;
  }
  store_partial<NT, RPT, BP>(a, tile == first_tile ? 0 : 1, acc);
  return true;
}

// Adds the partial sums of all contributors of a tile whose counter this workgroup completed, in workgroup order, and
// stores y. Contributors b_first..b_last: all but the first start inside the tile (slot 0); the first one used slot 1
// unless its range starts exactly at the tile. Loads are issued CH at a time so that they are in flight together.
template <int NT, int RPT, int BP>
__device__ __forceinline__ void reduce_tile(const GemmArgs& a, int64_t tile) {
  // loads in flight per thread: 16 contributors, at most 64 values (larger unrolls lengthen this rarely run, cold code,
  // and its registers count against the kernel's; the contributors are added in the same order whatever CH is)
  constexpr int CH = BP <= 4 ? 16 : 64 / BP;
  const int t = threadIdx.x;
  const int64_t R = int64_t(NT) * RPT;
  const int b_first = owner_of(a, int(tile) * a.steps);
  const int b_last = owner_of(a, int(tile + 1) * a.steps - 1);
  const int n_c = int(b_last - b_first + 1);
  const bool first_in_slot1 = first_unit(a, b_first) < int(tile) * a.steps;
  const char* pbase = reinterpret_cast<const char*>(a.partials);
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    const int r = t + NT * j;
    const int64_t row = tile * R + r;
    float sum[BP];
#pragma unroll
    for (int b = 0; b < BP; ++b) sum[b] = 0.f;
    for (int c0 = 0; c0 < n_c; c0 += CH) {
      float v[CH][BP];
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const int c = c0 + k;
        if constexpr (BP == 1) {
          // one batch row: contributors past n_c are not read (fewer loads in the launch's last microseconds)
          const int slot = (b_first + c) * 2 + ((c == 0 && first_in_slot1) ? 1 : 0);
          const char* src = pbase + int64_t(slot) * (R * 4);
          v[k][0] = c < n_c ? __hip_atomic_load(reinterpret_cast<const float*>(src + uint32_t(r * 4)),
                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                            : 0.f;
        } else {
          // several batch rows: past n_c the last contributor's slot is read again and its values are replaced by
          // zeros, so that the loads are unconditional and issued together (conditional loads become branches)
          const int cc = c < n_c ? c : n_c - 1;
          const int slot = (b_first + cc) * 2 + ((cc == 0 && first_in_slot1) ? 1 : 0);
          const char* src = pbase + int64_t(slot) * (BP * R * 4);
#pragma unroll
          for (int b = 0; b < BP; ++b)
            v[k][b] = __hip_atomic_load(reinterpret_cast<const float*>(src + uint32_t((b * R + r) * 4)),
                                        __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      if constexpr (BP > 1) {
#pragma unroll
        for (int k = 0; k < CH; ++k)
#pragma unroll
          for (int b = 0; b < BP; ++b)
            if (c0 + k >= n_c) v[k][b] = 0.f;
      }
#pragma unroll
      for (int k = 0; k < CH; ++k)
#pragma unroll
        for (int b = 0; b < BP; ++b) sum[b] += v[k][b];
    }
    if (row < a.M) {
#pragma unroll
      for (int b = 0; b < BP; ++b)
        if (b < a.B) store_y(a, b, row, sum[b]);
    }
  }
  if (t == 0) __hip_atomic_store(a.counters + tile * kCounterStride, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until every memory operation of the workgroup has completed, then publishes its pending tiles (at most two:
// its first and its last tile). Lanes 0 and 1 of the first wave bump the two counters with one instruction, so the two
// round trips are one; a counter that reaches the number of contributors makes this workgroup the one that reduces
// that tile.
// Ordering. The protocol relies on how gfx950 executes these instructions rather than on HIP's scoped acquire and
// release (an agent-scope acquire-release counter bump compiles to a write-back of the XCD's L2 before the atomic and
// an invalidate after it; on the 70B MLP layers that made every batch-1 call 7-10 us slower, 23 -> 30-33 us):
//   1. every partial sum is an agent-scope atomic store (global_store_dword ... sc1), which writes through the XCD's
//      L2 to the device's coherence point instead of leaving a line in a cache another XCD does not see;
//   2. s_waitcnt(0) waits until each of the thread's stores is acknowledged (on this gfx9-family ISA vmcnt counts
//      stores too), which for a write-through store happens once the data is at the coherence point; the barrier then
//      holds the workgroup until every thread has passed that wait;
//   3. the counter bump, a device-scope atomic read-modify-write, is issued after the barrier, so it is ordered after
//      every partial-sum store of the workgroup;
//   4. the reducing workgroup issues its partial-sum loads only after its own bump returned the completing count (the
//      loads are control-dependent on the returned value through the ballot and the barrier), and they are agent-scope
//      atomic loads (global_load_dword ... sc1), which do not hit stale lines of its CU's or XCD's caches.
template <int NT, int RPT, int BP>
__device__ __forceinline__ void publish_pending(const GemmArgs& a, int pending0, int pending1, int n_pending,
                                                int* s_flag) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (n_pending == 0) return;
  if (threadIdx.x < 64) {
    const int lane = int(threadIdx.x);
    const int tile = lane == 0 ? pending0 : pending1;
    bool last = false;
    if (lane < n_pending) {
      const uint32_t prev = __hip_atomic_fetch_add(a.counters + int64_t(tile) * kCounterStride, 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
      const int bf = owner_of(a, tile * a.steps);
      const int bl = owner_of(a, (tile + 1) * a.steps - 1);
      last = prev == uint32_t(bl - bf);
    }
    const uint64_t m = __ballot(last);
    if (lane == 0) *s_flag = int(m & 3u);
  }
  __syncthreads();
  const int flags = *s_flag;
  if (flags & 1) reduce_tile<NT, RPT, BP>(a, pending0);
  if (flags & 2) reduce_tile<NT, RPT, BP>(a, pending1);
}

// Read-only table entry with a wave-uniform index, through the constant address space so that it is a scalar load
// (its own counter): waiting for it never waits for the vector loads in flight.
__device__ __forceinline__ int32_t load_uniform_i32(const int32_t* p, int i) {
  return ((const __attribute__((address_space(4))) int32_t*)p)[i];
}

// Small-batch mu = 8 kernel (fluxbin_gemm_batch.hip): launches k_gemm_mu8_batch with n_groups groups of nb (2 or 4)
// batch rows and depth units of sign data requested ahead; with reduce2 (one group, depth 1) the split tiles are
// reduced by a second kernel instead of the tile counters; false if no instance exists.
// mx: kBigUnits for the instance staging up to that many units per workgroup (launch plan), else 0
bool launch_gemm_batch(const GemmArgs& a, int n_groups, int depth, int nb, bool reduce2, int mx, hipStream_t stream);

// Split tiles of a launch whose kernel stored every contributor's partial sums and skipped the tile counters, reduced
// by a second kernel over the whole chip (fluxbin_gemv.hip): bp padded batch rows, R rows per tile (a multiple of 256).
void launch_reduce_split(const GemmArgs& a, int bp, int R, hipStream_t stream);

// Matrix-core small-batch kernel (fluxbin_gemm_mfma.hip): 256-row tiles, partial sums padded to bpad (4, 8 or 16)
// batch rows, data requested depth (2 or 3) units ahead; with reduce2 (depth 2) the split tiles are reduced by a
// second kernel instead of the tile counters; false if no instance exists.
bool launch_gemm_mfma(const GemmArgs& a, int bpad, int mu, int depth, bool reduce2, hipStream_t stream);
// Row-complete small-batch kernel on the matrix cores (fluxbin_gemm_mfma_rows.hip): 16 rb rows per workgroup of
// 64 waves threads, bpad = 4 or 8 padded batch rows; false if no instance exists or the layer exceeds its limits.
bool launch_gemm_mfma_rows(const GemmArgs& a, int bpad, int mu, int waves, int rb, hipStream_t stream);

// Row-complete batch-1 kernel for layers with few rows (fluxbin_gemv_rows.hip): 16 rows per workgroup of `waves`
// (4, 8 or 16) wavefronts, every super-chunk of them, `depth` (2, 4 or 6) units requested ahead, fg (0, or 8 / 16 fine
// groups per salient chunk at mu = 8) as the batch-1 kernel's, no workspace; false if the layer is outside its limits
// (B = 1, N <= kRwMaxN, NSC <= min(waves, 8) * kRwSteps) or no instance exists.
// rb: 1 (16 rows per workgroup) or 2 (32 rows: each lane two rows; mu = 8 without fine groups)
bool launch_gemv_rows(const GemmArgs& a, int mu, int waves, int depth, int fg, int rb, hipStream_t stream);

}  // namespace fluxbin
