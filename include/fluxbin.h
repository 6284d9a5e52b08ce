/*
 * fluxbin.h - C ABI of the FluxBin LUT-GEMV hot path on AMD Instinct MI355X (gfx950).
 *
 * FluxBin (arXiv 2608.15602) stores a weight matrix W (M output rows x N input columns) as hybrid binary bases
 * (Sec. 3.1, Eqs. 3 and 9):
 *
 *   W-hat = sum_{k<Kb} (alpha_r^(k) alpha_c^(k)^T) .* B^(k)                       global bases
 *         + sum_{k<Ks} ((B_s^(k) .* Mask) .* (alpha_sr^(k) alpha_sc^(k)^T))          salient refinement
 *
 * with B in {-1,+1}, one row scale per (row, group of columns), one column scale per column, and the salient bases
 * restricted to a set I_sal of salient columns. The hot path computes Y = X W-hat^T for a batch of fp16 activation
 * rows X (Eq. 10) without dequantizing W: column scales are folded into the activations (Eq. 11), the salient columns
 * are remapped into a dense block (VCM, Eqs. 12-13), per mu-column sub-vector a table of all 2^mu signed partial sums
 * of (x * alpha_c) is built (LUT-BSF, Eq. 14), every mu-bit weight pattern indexes its table, and the row scales are
 * applied to the summed lookups (Eq. 15).
 *
 * Conventions for every entry point:
 *   - fp16 values are IEEE binary16 bit patterns passed as uint16_t.
 *   - Device pointers are HIP device memory of the current device; host pointers are ordinary host memory.
 *   - The caller owns every buffer. The library keeps no state between calls and allocates no device memory that
 *     outlives a call (fluxbin_pack with host inputs stages them in a temporary device buffer).
 *   - Device work is enqueued on the given stream and is asynchronous; no call synchronizes the device unless stated.
 *   - Every call validates its arguments on the host before any launch and returns a status; on failure nothing is
 *     launched and fluxbin_last_error_message() (thread-local) describes the problem.
 *   - Results are deterministic: the same inputs on the same device give bitwise identical outputs (no float atomics).
 *     The split of the work over workgroups (the launch plan), and with it the fp32 summation order, depends on the
 *     device's CU count and on the process-wide launch-plan tuning (fluxbin_tuning below: library defaults unless a
 *     caller changes them with fluxbin_set_tuning; the FLUXBIN_* environment variables named there are read once, at
 *     the library's first plan). Any plan gives the same product up to fp32 summation order; fluxbin_plan_query tells
 *     which kernel and plan a call would use.
 *   - Calls that share a workspace must not overlap in time (same stream, or ordered by the caller).
 */
#ifndef FLUXBIN_H_
#define FLUXBIN_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FLUXBIN_OK = 0,
  FLUXBIN_ERR_INVALID_ARG = 1,      /* null pointer, inconsistent sizes, unsorted salient set, ... */
  FLUXBIN_ERR_UNSUPPORTED = 2,      /* valid per the paper but outside what this library implements */
  FLUXBIN_ERR_BUFFER_TOO_SMALL = 3, /* packed buffer or workspace smaller than the query said */
  FLUXBIN_ERR_HIP = 4               /* a HIP runtime call failed; the message names it */
} fluxbin_status;

/* Static description of a status code. Never NULL. */
const char* fluxbin_status_string(fluxbin_status s);
/* Detail of the last failed call on this thread ("" if none). Valid until the next call on this thread. */
const char* fluxbin_last_error_message(void);

/*
 * Logical shape of one layer (paper notation, Sec. 3.1 and App. C.2).
 *   M    output channels (rows of W), 1 <= M <= 2^27 (the kernels address a row of a sign plane with 32-bit offsets).
 *   N    input channels (columns of W), 1 <= N <= 65535 (salient and activation indices are stored in 16 bits, as in
 *        App. C.2).
 *   Kb   global bases, 1..4.            Ks   salient bases, 0..4 (the paper uses Ks = Kb; the hybrid configs here 1).
 *   mu   LUT sub-vector length, 4 or 8 (Sec. 3.2 and App. E.2 use both; 8 is the paper's default).
 *   g_r  global row-scale group in columns: each row of each global base has its own scale for every run of g_r
 *        consecutive columns (Sec. 3.1; the 16*M*N/g storage term of App. C.2). A multiple of mu that divides 128
 *        (the paper's g = 64), a multiple of 128 (g = 128, 256), or g_r >= N (one per row).
 *   S    number of salient columns, 0..N (N_sal in the paper).
 *   g_s  salient row-scale group in VCM dense columns: one salient row scale per (row, salient base, group of g_s
 *        consecutive dense columns). The paper's structured selection (s salient columns in every block of g input
 *        columns, Sec. 3.1, Alg. FluxBin-Hybrid) with one salient row scale per (row, block) is g_s = s. Same rule as
 *        g_r (with S for N); ignored when S == 0 or Ks == 0.
 */
typedef struct {
  int64_t M, N;
  int32_t Kb, Ks;
  int32_t mu;
  int32_t reserved0;
  int64_t g_r;
  int64_t S;
  int64_t g_s;
} fluxbin_shape;

/*
 * Canonical (unpacked-layout) weights, read-only, all host or all device (inputs_on_device).
 *   signs      uint32 [Kb][M][W], W = ceil(N/32): bit t of word w is B^(k)[i, 32w+t] == +1 (a clear bit is -1, the
 *              (2b-1) map of Eq. 14). Bits past column N-1 are ignored.
 *   alpha_r    fp16 [Kb][M][G_r], G_r = ceil(N/g_r).
 *   alpha_c    fp16 [Kb][N].
 *   sal_idx    int32 [S], strictly increasing, each in [0, N) (I_sal, Eq. 8). May be NULL when S == 0.
 *   sal_signs  uint32 [Ks][M][W], FULL WIDTH like signs; only the bits of salient columns are read (B_s .* Mask).
 *   alpha_sr   fp16 [Ks][M][G_s], G_s = ceil(S/g_s).
 *   alpha_sc   fp16 [Ks][N], FULL WIDTH; the VCM gather (Eq. 13) is done at pack time.
 * Salient pointers may be NULL when S == 0 or Ks == 0.
 */
typedef struct {
  const uint32_t* signs;
  const uint16_t* alpha_r;
  const uint16_t* alpha_c;
  const int32_t* sal_idx;
  const uint32_t* sal_signs;
  const uint16_t* alpha_sr;
  const uint16_t* alpha_sc;
  int32_t inputs_on_device; /* 0: host pointers, 1: device pointers */
} fluxbin_weights;

/*
 * Packed layer: a POD descriptor of a caller-owned device buffer written by fluxbin_pack. It may be copied freely;
 * it stays valid as long as the buffer does. The same fields are stored in the buffer's 256-byte header, so the
 * buffer bytes alone are a serializable artifact (see fluxbin_layer_from_header).
 */
typedef struct {
  fluxbin_shape shape;
  void* d_base;         /* start of the packed device buffer */
  uint64_t bytes;       /* its size as returned by fluxbin_pack_query */
  uint32_t format_version;
  uint32_t reserved1;
  /* derived sizes (see PACKED FORMAT below) */
  int64_t Npad, Sv, NC, NSC, Mp, Gr, Gs, NRP;
  /* byte offsets of the sections from d_base */
  uint64_t off_signs, off_rscale, off_colscale, off_xidx, off_chunk_plane, off_sal_idx;
} fluxbin_layer;

/*
 * PACKED FORMAT (version 2). Written by fluxbin_pack, read by the GEMV kernels.
 *
 * Virtual columns. The global bases' columns and the salient bases' VCM dense columns (Def. VCM, Eq. 12: salient
 * column t of the dense block is input column I_sal[t]) are laid end to end in chunks of 128 columns:
 *   Npad = ceil(N/128)*128 and ncg = Npad/128 chunks per global base;
 *   Sv = ceil(S/128)*128 (0 if S == 0 or Ks == 0) and ncs = Sv/128 chunks per salient base;
 *   row scales per chunk and row: Gcg = 128/g_r for the global chunks when g_r < 128 and g_r < N ("fine" groups),
 *   else 1 ("coarse"); Gcs likewise from g_s and S for the salient chunks;
 *   ngcp = Kb*ncg global chunks, plus one inert separator chunk when Kb*ncg is odd, there is a salient part and
 *   Gcg != Gcs (so that the two chunks of a super-chunk share one scale layout);
 *   NC = ngcp + Ks*ncs chunks, NSC = ceil(NC/2) super-chunks of two chunks, NCP = 2*NSC (an odd NC gets one
 *   all-zero pad chunk), V = 128*NCP virtual columns; nfc = ngcp with a salient part, else NCP: chunks c >= nfc use
 *   the salient scale layout (Gcs), the others the global one (Gcg).
 * Chunk c < Kb*ncg is global base k = c / ncg, input columns ((c % ncg)*128 + r); chunk ngcp <= c < NC is salient
 * base k = (c - ngcp) / ncs, dense columns t = ((c - ngcp) % ncs)*128 + r, input column I_sal[t]. A virtual column
 * with no source (r past N, t past S, a pad chunk) has sign bit 0, column scale 0 and activation index 0xFFFF; it
 * contributes exactly zero.
 *
 * Sections (each starts at a multiple of 256 bytes, in this order after the 256-byte header):
 *   signs       [NSC][2][Mp][16] bytes, Mp = ceil(M/64)*64. Each 16-byte entry is one chunk of one row: 128 sign
 *               bits, split into P = 128/mu sub-vectors of mu bits (bit n of a sub-vector is its n-th column; set =
 *               +1), stored at rotated positions: with G the chunk's scales per row and n = P/G, position q of row i
 *               holds sub-vector ((floor(q/n) + floor(i/n)) mod G)*n + ((q mod n) + i) mod n (for G = 1 and G = P
 *               simply (q + i) mod P): the groups are rotated by floor(i/n) and the positions inside a group by i.
 *               mu = 8: slot h of super-chunk sc for row i holds chunk 2*sc + (h XOR [i mod 32 >= 16]); byte q is
 *               position q. mu = 4: slot h holds chunk 2*sc + h; nibble q (byte q/2, low nibble first) is position q.
 *               Rows i >= M are zero. (The rotation lets the 32 lanes of a half-wavefront read 32 different tables at
 *               the same step, so every LDS bank is hit once, and keeps each group's positions contiguous.)
 *   rscale      fp16 [NRP][Mp] planes. Global part (Pg planes): coarse, plane k*G_r + g holds alpha_r^(k)[:, g]
 *               (G_r = ceil(N/g_r), Pg = Kb*G_r); fine, chunk l of base k owns the Gcg planes from (k*ncg + l)*Gcg,
 *               read as [Mp][Gcg]: slot b of row i holds the scale of the chunk's group (b + floor(i/n)) mod Gcg,
 *               i.e. of the positions b*n .. b*n+n-1 (Pg = Kb*ncg*Gcg). Salient part, after the global planes: the
 *               same with alpha_sr, G_s = ceil(S/g_s), ncs, Gcs. Groups past the last one and rows >= M are zero.
 *   colscale    fp16 [V]: alpha_c^(k)[j] for global columns, alpha_sc^(k)[I_sal[t]] (= alpha_scd, Eq. 13) for salient
 *               dense columns, 0 for columns without a source.
 *   xidx        uint16 [V]: the input column j whose activation the virtual column reads, 0xFFFF for none.
 *   chunk_plane int32 [NCP]: first rscale plane of each chunk (a pad chunk has the planes of the chunk before it).
 *   sal_idx     uint16 [max(S,1)]: I_sal as 16-bit indices (App. C.2); a single 0 when S == 0.
 */
#define FLUXBIN_FORMAT_VERSION 2u
#define FLUXBIN_HEADER_BYTES 256u

/* Bytes of the packed buffer for a shape. Host only; validates the shape. */
fluxbin_status fluxbin_pack_query(const fluxbin_shape* shape, size_t* packed_bytes);

/*
 * Pack canonical weights into the device format (relayout of the sign planes, VCM extraction of the salient columns
 * and gather of their column scales, Eqs. 12-13). d_packed: caller-allocated device buffer of at least
 * fluxbin_pack_query bytes. Fills *out. With host inputs the call copies them to a temporary device buffer and
 * returns after the packing kernels complete; with device inputs it is asynchronous on `stream`.
 * The salient index set is validated on the host (host inputs) or copied to the host first (device inputs).
 */
fluxbin_status fluxbin_pack(const fluxbin_shape* shape, const fluxbin_weights* w, void* d_packed, size_t packed_bytes,
                            fluxbin_layer* out, hipStream_t stream);

/* Rebuild a layer descriptor from the 256-byte header of a packed buffer (copied to host memory by the caller) and
 * the device address where the packed bytes now live. Checks magic, version and sizes. */
fluxbin_status fluxbin_layer_from_header(const void* header_host, void* d_packed, size_t packed_bytes,
                                         fluxbin_layer* out);

/*
 * Workspace of one GEMV/GEMM call with batch B (1..8192): partial sums of output rows and one 32-bit counter per row
 * tile for split reductions, and for matrix-core launches of 16 or 32 rows the call's staged activations (one image
 * per super-chunk, rewritten by every call). Before its first use the workspace must be zero-filled
 * (fluxbin_workspace_init); every call leaves the counters at zero again. Calls sharing a workspace must not overlap
 * in time.
 * The counters sit in a region of the same size for every batch size of a layer, so calls of one layer with any
 * B may share one workspace (of the size queried for the largest B). A workspace used for another layer must first
 * be zero-filled again: the other layer's partial sums may cover this layer's counters.
 */
fluxbin_status fluxbin_workspace_query(const fluxbin_layer* layer, int32_t B, size_t* bytes);
fluxbin_status fluxbin_workspace_init(void* d_workspace, size_t bytes, hipStream_t stream);

/*
 * y = W-hat x for one fp16 activation vector (batch 1), Eqs. 10-15.
 *   d_x  fp16 [N] device.   d_y  [M] device, fp16 (y_is_fp32 = 0) or fp32 (y_is_fp32 = 1); must not alias d_x.
 * Sums are accumulated in fp32: x*alpha_c is exact in fp32, LUT entries and row sums are fp32, the fp16 output is
 * rounded to nearest even.
 */
fluxbin_status fluxbin_lut_gemv(const fluxbin_layer* layer, const uint16_t* d_x, void* d_y, int32_t y_is_fp32,
                                void* d_workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Y[b, :] = W-hat X[b, :] for b < B (1..8192). Up to T rows are one launch, which reads every packed sign word once
 * and uses it for all its rows (batch-independent reuse of the weights, Sec. 3.2 and App. E.2); larger batches run as
 * consecutive launches of T-row batch tiles (the last with the remaining rows), each its own launch plan, one after
 * another on the stream and sharing the workspace, so rows Tt..Tt+T-1 give the same y as a call on those rows alone.
 * T = 32 on layers with one row scale per chunk (matrix-core kernel), else 16; T = 1 (B launches of the batch-1
 * kernels) for B <= 8 on mu = 8 layers with 8 or 16 fine salient row-scale groups per chunk (the s16 / s8
 * configurations), unless the batch_tile tuning asks for 16. fluxbin_plan_query reports T as batch_tile_rows.
 * d_x fp16 with row stride ldx >= N (elements); d_y with row stride ldy >= M (elements of the output type). B = 1
 * gives the same result as fluxbin_lut_gemv.
 * Kernels: the LUT batch kernel (one set of tables per batch row; mu = 8, B <= 4 on layers with at least 2.25 (B = 2)
 * or 3.5 (B = 3, 4) 1024-row tiles of super-chunks per CU) and a matrix-core kernel (mu = 4, B > 4, or smaller
 * layers) that decodes the sign bits into fp16 +-alpha_c tiles and multiplies them with the activations on the MFMA
 * units (the products are exact in the fp32 accumulation, as in the LUT path; the row scale is applied per 128-column
 * chunk); on layers of 2048 to 4096 rows, or of at most 8192 rows with at most 88 super-chunks (on a 256-CU device),
 * at B <= 8 the matrix-core kernel runs row-complete (every super-chunk of 16 or 32 rows in one workgroup, no split
 * reduction). Other layers with fine row-scale groups (g_r or g_s below 128), and those above at B > 8, run the
 * generic LUT kernel for B >= 2. All are deterministic; their results differ only by fp32 summation order.
 */
fluxbin_status fluxbin_lut_gemm_smallbatch(const fluxbin_layer* layer, int32_t B, const uint16_t* d_x, int64_t ldx,
                                           void* d_y, int64_t ldy, int32_t y_is_fp32, void* d_workspace,
                                           size_t workspace_bytes, hipStream_t stream);

/*
 * fluxbin_lut_gemv for callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same product, launch plan and kernels as fluxbin_lut_gemv (bitwise the same
 * y), with the split-tile workspace taken from a static device array of FLUXBIN_NOALLOC_SCRATCH_BYTES that every
 * device the library runs on holds until the process ends. The call allocates nothing. Limits: M <= 64512 rows and
 * a launch plan needing at most FLUXBIN_NOALLOC_SCRATCH_BYTES of workspace, else FLUXBIN_ERR_UNSUPPORTED (nothing
 * launched). The first call on a device zero-fills that device's array on `stream`; every completed call leaves its
 * tile counters at zero again. All calls on one device share its array: calls that overlap in time on one device
 * (different streams, or different host threads without ordering) race and may return wrong results.
 */
#define FLUXBIN_NOALLOC_SCRATCH_BYTES (8u << 20)
fluxbin_status fluxbin_lut_gemv_noalloc(const fluxbin_layer* layer, const uint16_t* d_x, void* d_y, int32_t y_is_fp32,
                                        hipStream_t stream);

/*
 * Launch-plan tuning, for tests and measurements (the defaults are the library's measured choices). Process-wide: the
 * first plan made in a process initializes it from the environment variable named after each field (unset: default);
 * afterwards only fluxbin_set_tuning changes it (NULL restores the defaults). A plan takes one consistent copy, so
 * a change applies to the calls made after it returns. Fields and their defaults:
 *   nt             FLUXBIN_NT             batch-1 workgroup size 256 / 512 / 1024; 0: chosen by layer size
 *   min_units      FLUXBIN_MIN_UNITS      batch-1 minimum units per workgroup; -1: chosen by layer size
 *   blocks         FLUXBIN_BLOCKS         grid size target; 0: CU count times workgroups per CU
 *   blocks_per_cu  FLUXBIN_BLOCKS_PER_CU  workgroups per CU (1..8); 0: the kernel's occupancy
 *   depth          FLUXBIN_DEPTH          LUT kernels' units of sign data requested ahead (1..3); 0: 1
 *   mfma_depth     FLUXBIN_MFMA_DEPTH     matrix-core kernel's units requested ahead (2 or 3); 0: 2
 *   early          FLUXBIN_EARLY          batch-1 request order (1: signs before the activations); -1: by layer size
 *   rpt            FLUXBIN_RPT            generic kernel rows per thread (1, 2, 4); 0: chosen by layer size
 *   mfma           FLUXBIN_MFMA           small-batch kernel: 1 matrix cores, 0 LUT tables; -1: chosen by B and size
 *   generic        FLUXBIN_GENERIC        1: the generic kernel for every batch size
 *   mfma_r2        FLUXBIN_MFMA_R2        0: matrix-core split tiles reduced by tile counters, not a second kernel
 *   bat_r2         FLUXBIN_BAT_R2         0: LUT batch kernel split tiles reduced by tile counters
 *   rows           FLUXBIN_ROWS           batch 1: 1 the row-complete kernel where the layer allows it, 0 never;
 *                                         2 / 3 its 32- / 48-row workgroups (two / three rows per lane; mu = 8, on
 *                                         layers the kernel takes); -1: chosen by layer size
 *   batch_tile     FLUXBIN_BATCH_TILE     16: batch tiles of 16 rows on every layer; 0: 32 where the matrix-core
 *                                         kernel takes the layer
 *   mfma_rows      FLUXBIN_MFMA_ROWS      B = 2..8: 1 the row-complete matrix-core kernel wherever it fits, 0 never;
 *                                         -1: chosen by layer size
 *   align          FLUXBIN_ALIGN          split-tile kernels (batch-1, LUT batch, matrix-core): 0 workgroups over
 *                                         balanced unit ranges; -1 ranges aligned to row tiles where that fits one
 *                                         wave of workgroups; k > 0 aligned ranges, k workgroups per tile (clamped to
 *                                         what the unit cap and the tile allow)
 *   big_units      FLUXBIN_BIG_UNITS      batch-1 and LUT batch kernels: 0 at most 16 / 12 units per 1024-thread
 *                                         workgroup; -1 up to 24 where that fits a layer into one wave of workgroups
 */
typedef struct {
  int32_t nt, min_units, blocks, blocks_per_cu, depth, mfma_depth, early, rpt, mfma, generic, mfma_r2, bat_r2, rows,
      batch_tile, mfma_rows, align, big_units;
} fluxbin_tuning;
fluxbin_status fluxbin_get_tuning(fluxbin_tuning* out);
fluxbin_status fluxbin_set_tuning(const fluxbin_tuning* t);

/*
 * The launch plan a GEMV/GEMM call of batch B on this layer would use on the current device with the current tuning.
 *   kernel  0: batch-1 super-chunk kernel, 1: generic kernel, 2: LUT batch kernel (mu = 8), 3: matrix-core kernel,
 *           4: row-complete batch-1 kernel (layers with few rows; rows_per_tile 16, 32 or 48 rows per workgroup),
 *           5: row-complete matrix-core kernel (layers with few rows, B = 2..8).
 * Batches of more than batch_tile_rows rows (32 on layers the matrix-core kernel takes, else 16) run as batch_tiles
 * launches; the plan is then that of the full batch tiles, and workspace_bytes the call's workspace.
 * workgroups_per_tile > 0: the split-tile kernel's workgroups cover tile-aligned unit ranges, that many per row tile;
 * 0: balanced ranges over all units (or a kernel without split tiles). Host only apart
 * from reading the device's CU count; launches nothing.
 */
typedef struct {
  int32_t kernel, threads, rows_per_tile, depth, batch_groups, second_kernel_reduction, early, batch_tiles;
  int32_t batch_tile_rows, workgroups_per_tile;
  int64_t tiles, units, workgroups;
  uint64_t workspace_bytes;
} fluxbin_plan_info;
fluxbin_status fluxbin_plan_query(const fluxbin_layer* layer, int32_t B, fluxbin_plan_info* out);

/*
 * Test support. fluxbin_debug_indices writes the LUT index p read for every (chunk c < NCP, row i < M, sub-vector
 * u < 128/mu) into d_p[(c*M + i)*(128/mu) + u] (uint8), extracted from the packed signs by the same device code as the
 * kernels. fluxbin_unpack_canonical writes the global sign planes back in canonical form [Kb][M][W] (bits past N
 * zero) and, if d_dense_out is not NULL, the VCM dense salient planes [Ks][M][ceil(S/32)] (bit t of word w is dense
 * column 32w + t).
 */
fluxbin_status fluxbin_debug_indices(const fluxbin_layer* layer, uint8_t* d_p, hipStream_t stream);
fluxbin_status fluxbin_unpack_canonical(const fluxbin_layer* layer, uint32_t* d_signs_out, uint32_t* d_dense_out,
                                        hipStream_t stream);

/*
 * Measurement support (no result of the method). fluxbin_stream_probe reads the sign words and row scales of a packed
 * layer exactly as the split-tile batch-1 GEMV does (its launch plan, units, per-thread addresses and request depth,
 * also on layers whose default batch-1 plan is the row-complete kernel) but does no table work, giving the bandwidth
 * this access pattern can reach on the device; the benchmark reports the GEMV's bandwidth against it. d_sink (device,
 * at least 1024 bytes) receives meaningless checksums. Same validation and stream semantics as fluxbin_lut_gemv;
 * FLUXBIN_ERR_UNSUPPORTED for a layer the split-tile batch-1 kernel does not take (fine groups it has no instance
 * for, or the generic kernel forced by the tuning).
 */
fluxbin_status fluxbin_stream_probe(const fluxbin_layer* layer, uint32_t* d_sink, size_t sink_bytes,
                                    hipStream_t stream);

/*
 * Weight decomposition (the step that produces the hybrid bases; FluxBin Sec. 3.1), fp64 on the device.
 *
 * fluxbin_rc_decompose: RC_Decomp (App. algorithm "FluxBin Sub-routines"; Def. RC decomposition, Props. 3.2 and
 * 3.3) of X * mask, independently per block of g consecutive columns, into K binary bases
 * W^(k) = (alpha_r^(k) alpha_c^(k)^T) * B^(k) with one row scale per (row, block) and one column scale per column:
 * greedy residual initialization of every base (signs of the residual, column scale 1, one row-scale and one
 * column-scale least-squares update), then T rounds of (least-squares row and column scales of each base against
 * X * mask minus the other bases, Prop. 3.2; joint exhaustive sign search over the 2^K combinations per element,
 * first minimum in the order c = 0..2^K-1 with bit k of c set meaning +1, Prop. 3.3; signs times the mask).
 *   d_X        fp32 [M][N] row-major, device.        d_mask  uint8 [N] device (nonzero: column included), or NULL.
 *   K 1..4, T >= 0 rounds, g >= 1, eps >= 0 (the stability constant of Prop. 3.2).
 *   d_signs    uint32 [K][M][ceil(N/32)] device, canonical planes (bit t of word w: B[k][i][32w+t] == +1; columns
 *              off the mask have sign 0 and their bit clear).
 *   d_alpha_r  fp64 [K][M][ceil(N/g)] device.        d_alpha_c  fp64 [K][N] device (0 off the mask).
 *   d_ws       device workspace of fluxbin_rc_workspace_query bytes (the int8 signs during the rounds).
 *   Prior bases (optional, d_prior_signs NULL for none): X is replaced by X minus the approximation of Kp earlier bases
 *   (canonical ±1 bit planes [Kp][M][ceil(N/32)], row scales fp64 [Kp][M][ceil(N/gp)], column scales fp64 [Kp][N],
 *   all device), computed in fp64: the residual on which FluxBin-Hybrid decomposes the salient bases.
 * Asynchronous on `stream`; deterministic (fixed reduction orders, no atomics). Up to 2^36 elements.
 *
 * fluxbin_structural_search: Hessian-based column saliency (Def. in Sec. 3.1) with a diagonal inverse Hessian,
 * S_j = sum_i W_ij^2 / hinv_j^2 into d_scores (fp64 [N], device), and per block of g columns (g <= 1024, s <= g) the
 * s columns of largest saliency (equal scores: the smaller index first) into d_sal_idx (int32, device, increasing),
 * sum over blocks of min(s, block size) entries; if d_mask is not NULL also the column mask (uint8 [N], device: 1 for
 * a selected column).
 */
fluxbin_status fluxbin_rc_workspace_query(int64_t M, int64_t N, int32_t K, size_t* bytes);
fluxbin_status fluxbin_rc_decompose(const float* d_X, const uint8_t* d_mask, const uint32_t* d_prior_signs,
                                    const double* d_prior_alpha_r, const double* d_prior_alpha_c, int32_t Kp,
                                    int64_t gp, int64_t M, int64_t N, int32_t K, int32_t T, int64_t g, double eps,
                                    uint32_t* d_signs, double* d_alpha_r, double* d_alpha_c, void* d_ws,
                                    size_t ws_bytes, hipStream_t stream);
fluxbin_status fluxbin_structural_search(const float* d_W, const double* d_hinv_diag, int64_t M, int64_t N,
                                         int64_t g, int64_t s, double* d_scores, int32_t* d_sal_idx, uint8_t* d_mask,
                                         hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FLUXBIN_H_ */
