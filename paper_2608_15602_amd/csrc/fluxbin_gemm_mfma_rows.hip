// Small-batch (B = 2..8) product of libfluxbin on the gfx950 matrix cores for layers with few rows: row-complete
// workgroups, so that no partial sum crosses a workgroup.
//
// What is computed is the matrix-core kernel's contraction (fluxbin_gemm_mfma.hip: Eqs. 10-11 and 15 with the inner
// sums of a chunk as v_mfma_f32_16x16x32_f16 over exact fp16 operands, A = -s * colscale, B = x, the row scale applied
// once per 128-column chunk, negated). That kernel splits every 256-row tile's super-chunks over several workgroups and
// reduces the split tiles with a second kernel: on a layer of a few thousand rows the call is then mostly start-up,
// the partial-sum stores, the second launch and its loads (4096 x 4096 at B = 2..8: about 11 us, twice the batch-1
// row-complete kernel). Here a workgroup owns RB 16-row MFMA blocks and every super-chunk of them: its W wavefronts take
// every W-th super-chunk, and add their accumulators through LDS in wavefront order at the end.
//
// Activations. A chunk's B operands depend only on the x columns it reads: global chunks of all bases read the same
// column block (chunk c < ngc reads the columns of chunk c mod ncg), the other chunks (salient, separator, padding)
// their own gathered columns. At the start the workgroup stages one activation block per distinct column block, in the
// order the MFMA lanes read it: block (column block, group g, K step q) holds for batch row b the four fp16 pairs
// (x[b][xidx[v]], x[b][xidx[v + 16]]), v = 32 g + 4 q + k, at dwords 4 b + k (zero for a column with no source and rows
// >= B), and the signed column-scale pairs of every chunk (the A operand before its sign bits). Gathered per workgroup
// these took a dependent round trip per element (4096 x 4096: 10.7 us at B = 2 against 6.0 without them); instead a
// first kernel writes them once per call to an image in the workspace, which every workgroup copies into LDS with
// LDS-direct loads, waited for with vmcnt before the first barrier while its first sign requests stay in flight.
// MFMA lanes of batch columns >= BP read past their block: those columns of the product are never stored, and each
// column of an MFMA result depends on that column of its B operand only. The sign entries of a unit pass through the wavefront's own LDS
// scratch to the MFMA lanes, and are decoded as in the split-tile kernel (the words of one row's two chunks shifted
// together by one 64-bit shift).
#include <hip/hip_runtime.h>

#include "fluxbin_device.h"

namespace fluxbin {

namespace {

typedef _Float16 mr_half8 __attribute__((ext_vector_type(8)));
typedef float mr_float4 __attribute__((ext_vector_type(4)));
typedef unsigned int mr_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int mr_u32x2 __attribute__((ext_vector_type(2)));

// dwords per (column block, group, K step) activation block: BP rows x 4 pairs and 4 dwords of padding
// (mfma_rows_lds_bytes leaves 64 dwords after the last block: lanes of batch columns >= BP read up to 60 past it)
template <int BP> constexpr int mr_bstride() { return 4 * BP + 4; }

// Requested data of one unit for one lane: the 16-byte entry it loads (lane l < 32 RB: row l & 15 of row block
// l >> 5, chunk (l >> 4) & 1; other lanes load nothing) and the fp16 row scales of its MFMA output rows (rows
// 4g..4g+3 of each row block, g = l >> 4) of both chunks.
template <int RB>
struct MrRegs {
  mr_u32x4 e;
  mr_u32x2 rs[2][RB];
};

struct MrLane {
  int t, lane, w, r16, g;
  bool loads;          // the lane loads a 16-byte entry
  uint32_t voff_e;     // its entry in super-chunk 0: slot and row
  uint32_t scr_e;      // dword offset of its entry in a unit's scratch: (h RB + rb) 64 + 4 r
  uint32_t voff_rs;    // (row0 + 4 g) * 2: its output rows in a row-scale plane (row block rb adds 32 bytes)
  uint32_t wa[2][2];   // scratch offsets of the two words holding canonical bits 32g..32g+31 (by row-block parity)
  uint32_t sh;         // funnel shift
};

// 64-bit left shift by a constant, as one v_lshlrev_b64 (the compiler would split it into two 32-bit shifts).
__device__ __forceinline__ uint64_t mr_shl64(uint64_t v, uint32_t s) {
  uint64_t r;
  asm("v_lshlrev_b64 %0, %1, %2" : "=v"(r) : "s"(s), "v"(v));
  return r;
}

template <int RB>
__device__ __forceinline__ void mr_issue(const GemmArgs& a, const __amdgpu_buffer_rsrc_t& rsig,
                                         const __amdgpu_buffer_rsrc_t& rrs, const MrLane& ln, int sc, int p0, int p1,
                                         MrRegs<RB>& u) {
  if (ln.loads) u.e = __builtin_bit_cast(mr_u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsig, int(ln.voff_e),
                                                                                          2 * sc * a.Mp * 16, 0));
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    u.rs[0][rb] = __builtin_bit_cast(mr_u32x2, __builtin_amdgcn_raw_buffer_load_b64(rrs, int(ln.voff_rs) + 32 * rb,
                                                                                     p0 * a.Mp * 2, 0));
    u.rs[1][rb] = __builtin_bit_cast(mr_u32x2, __builtin_amdgcn_raw_buffer_load_b64(rrs, int(ln.voff_rs) + 32 * rb,
                                                                                     p1 * a.Mp * 2, 0));
  }
}

// One unit (super-chunk sc) into the accumulators. scr: the wavefront's scratch of the unit; cs: column-scale pairs
// (64 dwords per chunk: group g, K step q, pair k at 16 g + 4 q + k); xp: activation blocks; blk0, blk1: the column
// blocks of the unit's two chunks.
template <int BP, int RB, int MU>
__device__ __forceinline__ void mr_unit(const uint32_t* scr, const uint32_t* cs, const uint32_t* xp, int sc, int blk0,
                                        int blk1, const MrLane& ln, int par0, const MrRegs<RB>& u,
                                        float (&acc)[RB][4]) {
  constexpr int BS = mr_bstride<BP>();
  uint64_t w2[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const bool odd = MU == 4 && ((par0 + rb) & 1) != 0;   // selected, not indexed: no private array
    const uint32_t wa0 = odd ? ln.wa[1][0] : ln.wa[0][0];
    const uint32_t wa1 = odd ? ln.wa[1][1] : ln.wa[0][1];
    uint32_t w[2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
      w[h] = __builtin_amdgcn_alignbit(scr[(h * RB + rb) * 64 + wa1], scr[(h * RB + rb) * 64 + wa0], ln.sh);
    w2[rb] = (uint64_t(w[1]) << 32) | w[0];   // chunk 0 low, chunk 1 high: one shift serves both
  }
  const uint32_t* csh[2] = {cs + (2 * sc) * 64 + 16 * ln.g, cs + (2 * sc + 1) * 64 + 16 * ln.g};
  const uint32_t* xph[2] = {xp + (blk0 * 16 + 4 * ln.g) * BS + 4 * ln.r16, xp + (blk1 * 16 + 4 * ln.g) * BS + 4 * ln.r16};
  mr_float4 tmp[RB][2];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    mr_u32x4 ac[2], bx[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      ac[h] = *reinterpret_cast<const mr_u32x4*>(csh[h] + 4 * q);
      bx[h] = *reinterpret_cast<const mr_u32x4*>(xph[h] + q * BS);
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      mr_u32x4 av0, av1;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint64_t sft = mr_shl64(w2[rb], uint32_t(15 - (4 * q + k)));
        av0[k] = (uint32_t(sft) & 0x80008000u) ^ ac[0][k];
        av1[k] = (uint32_t(sft >> 32) & 0x80008000u) ^ ac[1][k];
      }
      const mr_float4 c0 = q == 0 ? mr_float4{0.f, 0.f, 0.f, 0.f} : tmp[rb][0];
      const mr_float4 c1 = q == 0 ? mr_float4{0.f, 0.f, 0.f, 0.f} : tmp[rb][1];
      tmp[rb][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mr_half8, av0),
                                                          __builtin_bit_cast(mr_half8, bx[0]), c0, 0, 0, 0);
      tmp[rb][1] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(mr_half8, av1),
                                                          __builtin_bit_cast(mr_half8, bx[1]), c1, 0, 0, 0);
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      acc[rb][0] = fmaf(-h2f(uint16_t(u.rs[h][rb][0])), tmp[rb][h][0], acc[rb][0]);
      acc[rb][1] = fmaf(-h2f(uint16_t(u.rs[h][rb][0] >> 16)), tmp[rb][h][1], acc[rb][1]);
      acc[rb][2] = fmaf(-h2f(uint16_t(u.rs[h][rb][1])), tmp[rb][h][2], acc[rb][2]);
      acc[rb][3] = fmaf(-h2f(uint16_t(u.rs[h][rb][1] >> 16)), tmp[rb][h][3], acc[rb][3]);
    }
}

// LDS address (bytes) of a pointer into the workgroup's LDS.
__device__ __forceinline__ uint32_t mr_lds_addr(const uint32_t* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const uint32_t*)(p)));
}

// One 1 KB LDS-direct request: lane l's 16 bytes at src (per lane) land at dst + 4 l (dst wave-uniform). M0 holds the
// request's LDS address (one wait state between its write and the load). Written as an instruction: with the compiler's
// builtin the compiler would drain every outstanding load before each later barrier.
__device__ __forceinline__ void mr_copy16(const uint32_t* src, uint32_t* dst) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(mr_lds_addr(dst)), "v"(src)
               : "memory");
}

// The call's staging image (first of the two kernels; one thread per image dword, mfma_rows_image_dwords in all):
// column-scale pairs of every chunk (dword c 64 + 16 g + 4 q + k: the signed column scales of columns 32 g + 4 q + k
// and that + 16 of chunk c), then the activation blocks (block (column block, g, q) at (blk 16 + 4 g + q) BS: for batch
// row b < B the fp16 pairs (x[b][xidx[v]], x[b][xidx[v + 16]]) of v = 32 g + 4 q + k of a chunk reading the column
// block, at 4 b + k; zero for a column with no source, rows >= B, padding), then zeros to a whole 1 KB.
template <int BP>
__global__ void __launch_bounds__(256) k_mr_image(GemmArgs a) {
  constexpr int BS = mr_bstride<BP>();
  const int nblk = a.ncg + (a.NCP - a.ngc);
  const int d = blockIdx.x * 256 + threadIdx.x;
  uint32_t v = 0u;
  if (d < a.NCP * 64) {
    const int c = d >> 6, e = d & 63;
    const int col = c * 128 + 32 * (e >> 4) + (e & 15);
    v = uint32_t(a.colscale[col]) | (uint32_t(a.colscale[col + 16]) << 16);
  } else if (d < a.NCP * 64 + nblk * 16 * BS) {
    const int dd = d - a.NCP * 64;
    const int blk = dd / (16 * BS);
    const int rem = dd - blk * (16 * BS);
    const int gq = rem / BS, o = rem - gq * BS;
    const int b = o >> 2;
    if (o < 4 * BP && b < a.B) {
      const int csrc = blk < a.ncg ? blk : a.ngc + (blk - a.ncg);   // a chunk reading this column block
      const int col = csrc * 128 + 32 * (gq >> 2) + 4 * (gq & 3) + (o & 3);
      const uint32_t i0 = a.xidx[col], i1 = a.xidx[col + 16];
      const uint16_t* xr = a.x + int64_t(b) * a.ldx;
      v = (i0 == 0xFFFFu ? 0u : uint32_t(xr[i0])) | ((i1 == 0xFFFFu ? 0u : uint32_t(xr[i1])) << 16);
    }
  }
  if (d < int(mfma_rows_image_dwords(a.NCP, nblk, BP))) a.img[d] = v;
}

template <int BP, int MU, int W, int RB, int D>
struct MrKernel {
  struct Ctx {
    __amdgpu_buffer_rsrc_t rsig, rrs;
    const int* s_plane;
    const int* s_blk;
    const uint32_t* cs;
    const uint32_t* xp;
    uint32_t* scr;   // the wavefront's scratch: two units of 2 RB 64 dwords
    int n;           // units of this wavefront: super-chunks w, w + W, ...
    int par0;        // parity of the workgroup's first row block (mu = 4 rotation)
  };

  // Unit K of the wavefront, register set K mod (D + 1): request unit K+D, stage unit K+1's entries, multiply unit K.
  template <int K>
  __device__ static __forceinline__ void step(const GemmArgs& a, const Ctx& cx, const MrLane& ln,
                                              MrRegs<RB> (&ur)[D + 1], float (&acc)[RB][4]) {
    if constexpr (K < kMrSteps) {
      if (K >= cx.n) return;
      if (K + D < cx.n) {
        const int scn = ln.w + (K + D) * W;
        mr_issue<RB>(a, cx.rsig, cx.rrs, ln, scn, __builtin_amdgcn_readfirstlane(cx.s_plane[2 * scn]),
                     __builtin_amdgcn_readfirstlane(cx.s_plane[2 * scn + 1]), ur[(K + D) % (D + 1)]);
      }
      if (K + 1 < cx.n && ln.loads)
        *reinterpret_cast<mr_u32x4*>(cx.scr + ((K + 1) & 1) * (2 * RB * 64) + ln.scr_e) = ur[(K + 1) % (D + 1)].e;
      const int sc = ln.w + K * W;
      const int blk0 = __builtin_amdgcn_readfirstlane(cx.s_blk[2 * sc]);
      const int blk1 = __builtin_amdgcn_readfirstlane(cx.s_blk[2 * sc + 1]);
      mr_unit<BP, RB, MU>(cx.scr + (K & 1) * (2 * RB * 64), cx.cs, cx.xp, sc, blk0, blk1, ln, cx.par0,
                          ur[K % (D + 1)], acc);
      step<K + 1>(a, cx, ln, ur, acc);
    }
  }
};

template <int BP, int MU, int W, int RB, int D>
__global__ void __launch_bounds__(64 * W) k_gemm_mfma_rows(GemmArgs a) {
  using K = MrKernel<BP, MU, W, RB, D>;
  constexpr int NT = 64 * W;
  constexpr int BS = mr_bstride<BP>();
  // dynamic: column-scale pairs (NCP x 64 dwords), then the activation blocks (NBLK x 16 x BS dwords + slack)
  extern __shared__ __attribute__((aligned(16))) uint32_t mr_dyn[];
  // sign scratch, two units per wavefront; at the end each wavefront's accumulators (W RB 256 floats: the same size)
  __shared__ __attribute__((aligned(16))) uint32_t scr_all[W * 2 * 2 * RB * 64];
  float* s_red = reinterpret_cast<float*>(scr_all);
  __shared__ int s_plane[2 * W * kMrSteps];
  __shared__ int s_blk[2 * W * kMrSteps];

  MrLane ln;
  ln.t = threadIdx.x;
  ln.lane = ln.t & 63;
  ln.w = __builtin_amdgcn_readfirstlane(ln.t >> 6);
  ln.r16 = ln.lane & 15;
  ln.g = ln.lane >> 4;
  const int row0 = int(blockIdx.x) * 16 * RB;   // rows row0 .. row0 + 16 RB - 1 < Mp (Mp: a multiple of 64)
  {
    const int rb = ln.lane >> 5, h = (ln.lane >> 4) & 1;
    ln.loads = ln.lane < 32 * RB;
    const int row = row0 + 16 * (ln.loads ? rb : 0) + ln.r16;
    // mu = 8 stores the two chunks of a super-chunk swapped for rows with i mod 32 >= 16
    const int slot = MU == 8 ? (h ^ ((row >> 4) & 1)) : h;
    ln.voff_e = uint32_t(slot * a.Mp * 16 + row * 16);
    ln.scr_e = uint32_t((h * RB + (ln.loads ? rb : 0)) * 64 + 4 * ln.r16);
  }
  ln.voff_rs = uint32_t((row0 + 4 * ln.g) * 2);
  // words of a row's entry that hold canonical bits 32g..32g+31: they start at stored bit (32g - R) mod 128, R = 8 r
  // (mu = 8) or 4 r plus 64 for odd 16-row blocks (mu = 4)
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

  typename K::Ctx cx;
  cx.n = ln.w < a.NSC ? (a.NSC - 1 - ln.w) / W + 1 : 0;
  cx.par0 = (row0 >> 4) & 1;
  const int nblk = a.ncg + (a.NCP - a.ngc);
  uint32_t* cs = mr_dyn;
  uint32_t* xp = mr_dyn + a.NCP * 64;
  cx.cs = cs;
  cx.xp = xp;
  cx.s_plane = s_plane;
  cx.s_blk = s_blk;
  cx.scr = scr_all + ln.w * (2 * 2 * RB * 64);

  // Staging: the chunk tables, then the call's image of column-scale pairs and activation blocks (k_mr_image), copied
  // LDS-direct (16 bytes per lane straight to LDS, 1 KB requests dealt round-robin to the wavefronts).
  for (int c = ln.t; c < a.NCP; c += NT) {
    s_plane[c] = a.chunk_plane[c];
    s_blk[c] = c < a.ngc ? c % a.ncg : a.ncg + (c - a.ngc);
  }
  {
    const int nreq = int(mfma_rows_image_dwords(a.NCP, nblk, BP) / 256);
    const uint32_t* src = a.img + 4 * ln.lane;
    for (int r = ln.w; r < nreq; r += W) mr_copy16(src + 256 * r, mr_dyn + 256 * r);
  }

  cx.rsig = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(a.signs), 0, a.NCP * a.Mp * 16, 0x00020000);
  cx.rrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(a.rscale), 0, 0x7FFFFFFF, 0x00020000);
  // units 0..D-1, requested by every wavefront (clamped to the last super-chunk where it has fewer), so that each has
  // issued exactly D (1 + 2 RB) vector loads after its image copies
  MrRegs<RB> ur[D + 1];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    const int sc = ln.w + k * W < a.NSC ? ln.w + k * W : a.NSC - 1;
    mr_issue<RB>(a, cx.rsig, cx.rrs, ln, sc, load_uniform_i32(a.chunk_plane, 2 * sc),
                 load_uniform_i32(a.chunk_plane, 2 * sc + 1), ur[k]);
  }
  float acc[RB][4];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[rb][v] = 0.f;
  if (cx.n > 0 && ln.loads) *reinterpret_cast<mr_u32x4*>(cx.scr + ln.scr_e) = ur[0].e;
  // all but the last D (1 + 2 RB) vector memory operations (those sign and row-scale requests) have completed: the
  // wavefront's image copies have landed
  static_assert(D == 2 && (RB == 1 || RB == 2), "vmcnt below counts two units of 1 + 2 RB requests");
  if constexpr (RB == 1)
    asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(10)" ::: "memory");
  __syncthreads();   // staging done
  K::template step<0>(a, cx, ln, ur, acc);

  // the wavefronts' accumulators in wavefront order: lane (b, g) holds rows 4g..4g+3 of each row block, batch row b;
  // wavefront w writes its own scratch, which it has finished reading
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int v = 0; v < 4; ++v) s_red[((ln.w * RB + rb) * 16 + 4 * ln.g + v) * 16 + ln.r16] = acc[rb][v];
  __syncthreads();
  for (int i = ln.t; i < RB * 16 * 16; i += NT) {
    const int b = i & 15, rr = i >> 4;   // rr = 16 rb + r
    if (b >= a.B) continue;
    float y = s_red[rr * 16 + b];
#pragma unroll
    for (int w = 1; w < W; ++w) y += s_red[(w * RB * 16 + rr) * 16 + b];
    const int64_t row = int64_t(row0) + rr;
    if (row < a.M) store_y(a, b, row, y);
  }
}

template <int BP, int W, int RB>
bool launch_mr(const GemmArgs& a, int mu, hipStream_t stream) {
  const dim3 grid(unsigned((a.M + 16 * RB - 1) / (16 * RB))), block(64 * W);
  const int64_t nblk = a.ncg + (a.NCP - a.ngc);
  const unsigned lds = unsigned(mfma_rows_lds_bytes(a.NCP, nblk, BP));
  if (mu != 8 && mu != 4) return false;
  hipLaunchKernelGGL((k_mr_image<BP>), dim3(unsigned(mfma_rows_image_dwords(a.NCP, nblk, BP) / 256)), dim3(256), 0,
                     stream, a);
  if (mu == 8)
    hipLaunchKernelGGL((k_gemm_mfma_rows<BP, 8, W, RB, 2>), grid, block, lds, stream, a);
  else if (mu == 4)
    hipLaunchKernelGGL((k_gemm_mfma_rows<BP, 4, W, RB, 2>), grid, block, lds, stream, a);
  else
    return false;
  return true;
}

template <int BP>
bool launch_mr_bp(const GemmArgs& a, int mu, int waves, int rb, hipStream_t stream) {
  if (waves == 8 && rb == 1) return launch_mr<BP, 8, 1>(a, mu, stream);
  if (waves == 8 && rb == 2) return launch_mr<BP, 8, 2>(a, mu, stream);
  if (waves == 16 && rb == 1) return launch_mr<BP, 16, 1>(a, mu, stream);
  if (waves == 16 && rb == 2) return launch_mr<BP, 16, 2>(a, mu, stream);
  return false;
}

}  // namespace

bool launch_gemm_mfma_rows(const GemmArgs& a, int bpad, int mu, int waves, int rb, hipStream_t stream) {
  if (a.B < 1 || a.B > bpad || a.NSC > waves * kMrSteps) return false;
  if (bpad == 4) return launch_mr_bp<4>(a, mu, waves, rb, stream);
  if (bpad == 8) return launch_mr_bp<8>(a, mu, waves, rb, stream);
  return false;
}

}  // namespace fluxbin
