// Host side of libfluxbin: argument validation, format sizes, launch planning and the C ABI entry points.
// Every check runs before any HIP call so that invalid input never reaches a kernel.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "fluxbin_internal.h"

namespace fluxbin {

static thread_local char g_msg[512] = "";

void clear_error() { g_msg[0] = 0; }

fluxbin_status fail(fluxbin_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return s;
}

fluxbin_status hip_fail(int err, const char* what) {
  return fail(FLUXBIN_ERR_HIP, "%s failed: %s", what, hipGetErrorString(static_cast<hipError_t>(err)));
}

int device_cu_count() {
  static std::mutex mu;
  static int cache[64] = {};   // per device index (no allocation: fluxbin_lut_gemv_noalloc plans through this)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return -1;
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return -1;
    cache[dev] = n;
  }
  return cache[dev];
}

static fluxbin_status check_shape(const fluxbin_shape* s) {
  if (!s) return fail(FLUXBIN_ERR_INVALID_ARG, "shape is NULL");
  // M <= 2^27 keeps every byte offset of a row inside the two sign planes of a super-chunk below 2^32
  if (s->M < 1 || s->M > (int64_t(1) << 27))
    return fail(FLUXBIN_ERR_INVALID_ARG, "M = %lld out of range [1, 2^27]", (long long)s->M);
  if (s->N < 1) return fail(FLUXBIN_ERR_INVALID_ARG, "N = %lld must be >= 1", (long long)s->N);
  if (s->N > 65535)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "N = %lld exceeds 65535 (16-bit column indices)", (long long)s->N);
  if (s->Kb < 1 || s->Kb > 4) return fail(FLUXBIN_ERR_INVALID_ARG, "Kb = %d out of range [1, 4]", s->Kb);
  if (s->Ks < 0 || s->Ks > 4) return fail(FLUXBIN_ERR_INVALID_ARG, "Ks = %d out of range [0, 4]", s->Ks);
  if (s->mu < 1 || s->mu > 16) return fail(FLUXBIN_ERR_INVALID_ARG, "mu = %d out of range", s->mu);
  if (s->mu != 4 && s->mu != 8) return fail(FLUXBIN_ERR_UNSUPPORTED, "mu = %d (supported: 4, 8)", s->mu);
  if (s->g_r < 1) return fail(FLUXBIN_ERR_INVALID_ARG, "g_r = %lld must be >= 1", (long long)s->g_r);
  if (s->g_r < s->N && s->g_r % s->mu != 0)
    return fail(FLUXBIN_ERR_INVALID_ARG, "g_r = %lld must hold whole sub-vectors of mu = %d", (long long)s->g_r, s->mu);
  if (s->g_r < s->N && s->g_r % kChunk != 0 && kChunk % s->g_r != 0)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "g_r = %lld: supported are divisors of 128, multiples of 128, or g_r >= N",
                (long long)s->g_r);
  if (s->S < 0 || s->S > s->N)
    return fail(FLUXBIN_ERR_INVALID_ARG, "S = %lld out of range [0, N]", (long long)s->S);
  if (s->S > 0 && s->Ks > 0) {
    if (s->g_s < 1) return fail(FLUXBIN_ERR_INVALID_ARG, "g_s = %lld must be >= 1", (long long)s->g_s);
    if (s->g_s < s->S && s->g_s % s->mu != 0)
      return fail(FLUXBIN_ERR_INVALID_ARG, "g_s = %lld must hold whole sub-vectors of mu = %d", (long long)s->g_s,
                  s->mu);
    if (s->g_s < s->S && s->g_s % kChunk != 0 && kChunk % s->g_s != 0)
      return fail(FLUXBIN_ERR_UNSUPPORTED, "g_s = %lld: supported are divisors of 128, multiples of 128, or g_s >= S",
                  (long long)s->g_s);
  }
  return FLUXBIN_OK;
}

static void fill_layer(const fluxbin_shape& s, void* d_base, uint64_t bytes, fluxbin_layer* L) {
  const Derived d = derive(s);
  const Offsets o = offsets(s, d);
  std::memset(L, 0, sizeof(*L));
  L->shape = s;
  L->d_base = d_base;
  L->bytes = bytes;
  L->format_version = FLUXBIN_FORMAT_VERSION;
  L->Npad = d.Npad;
  L->Sv = d.Sv;
  L->NC = d.NC;
  L->NSC = d.NSC;
  L->Mp = d.Mp;
  L->Gr = d.Gr;
  L->Gs = d.Gs;
  L->NRP = d.NRP;
  L->off_signs = o.signs;
  L->off_rscale = o.rscale;
  L->off_colscale = o.colscale;
  L->off_xidx = o.xidx;
  L->off_chunk_plane = o.chunk_plane;
  L->off_sal_idx = o.sal_idx;
}

static fluxbin_status check_layer(const fluxbin_layer* L) {
  if (!L) return fail(FLUXBIN_ERR_INVALID_ARG, "layer is NULL");
  if (L->format_version != FLUXBIN_FORMAT_VERSION)
    return fail(FLUXBIN_ERR_INVALID_ARG, "layer format version %u (expected %u)", L->format_version,
                FLUXBIN_FORMAT_VERSION);
  if (!L->d_base) return fail(FLUXBIN_ERR_INVALID_ARG, "layer has no device buffer");
  fluxbin_status st = check_shape(&L->shape);
  if (st != FLUXBIN_OK) return st;
  fluxbin_layer ref;
  fill_layer(L->shape, L->d_base, L->bytes, &ref);
  if (std::memcmp(&ref, L, sizeof(ref)) != 0)
    return fail(FLUXBIN_ERR_INVALID_ARG, "layer descriptor is inconsistent with its shape");
  if (L->bytes < offsets(L->shape, derive(L->shape)).total)
    return fail(FLUXBIN_ERR_BUFFER_TOO_SMALL, "layer buffer is smaller than its format needs");
  return FLUXBIN_OK;
}

// ---- launch-plan tuning: read from the FLUXBIN_* environment once per process, then only changed through
// fluxbin_set_tuning (tests and measurements); every plan takes one consistent snapshot ----
static fluxbin_tuning tuning_defaults() {
  fluxbin_tuning t;
  std::memset(&t, 0, sizeof(t));
  t.nt = 0;
  t.min_units = -1;
  t.blocks = 0;
  t.blocks_per_cu = 0;
  t.depth = 0;
  t.mfma_depth = 0;
  t.early = -1;
  t.rpt = 0;
  t.mfma = -1;
  t.generic = 0;
  t.mfma_r2 = 1;
  t.bat_r2 = 1;
  t.rows = -1;
  t.batch_tile = 0;
  t.mfma_rows = -1;
  t.align = -1;
  t.big_units = -1;
  return t;
}

static int env_int(const char* name, int dflt) {
  const char* v = std::getenv(name);
  if (!v || !*v) return dflt;
  return std::atoi(v);
}

static std::mutex g_tuning_mu;
static bool g_tuning_init = false;
static fluxbin_tuning g_tuning;

static void tuning_init_locked() {
  if (g_tuning_init) return;
  fluxbin_tuning t = tuning_defaults();
  t.nt = env_int("FLUXBIN_NT", t.nt);
  t.min_units = env_int("FLUXBIN_MIN_UNITS", t.min_units);
  t.blocks = env_int("FLUXBIN_BLOCKS", t.blocks);
  t.blocks_per_cu = env_int("FLUXBIN_BLOCKS_PER_CU", t.blocks_per_cu);
  t.depth = env_int("FLUXBIN_DEPTH", t.depth);
  t.mfma_depth = env_int("FLUXBIN_MFMA_DEPTH", t.mfma_depth);
  t.early = env_int("FLUXBIN_EARLY", t.early);
  t.rpt = env_int("FLUXBIN_RPT", t.rpt);
  t.mfma = env_int("FLUXBIN_MFMA", t.mfma);
  t.generic = env_int("FLUXBIN_GENERIC", t.generic);
  t.mfma_r2 = env_int("FLUXBIN_MFMA_R2", t.mfma_r2);
  t.bat_r2 = env_int("FLUXBIN_BAT_R2", t.bat_r2);
  t.rows = env_int("FLUXBIN_ROWS", t.rows);
  t.batch_tile = env_int("FLUXBIN_BATCH_TILE", t.batch_tile);
  t.mfma_rows = env_int("FLUXBIN_MFMA_ROWS", t.mfma_rows);
  t.align = env_int("FLUXBIN_ALIGN", t.align);
  t.big_units = env_int("FLUXBIN_BIG_UNITS", t.big_units);
  g_tuning = t;
  g_tuning_init = true;
}

static fluxbin_tuning tuning_snapshot() {
  std::lock_guard<std::mutex> lock(g_tuning_mu);
  tuning_init_locked();
  return g_tuning;
}

// Small-batch kernel choice (both kernels reduce split tiles with the second kernel). The matrix-core kernel's cost per
// sign bit (decode) is the same for every B <= 16 (B <= 4 share one padded instance); the mu = 8 LUT batch kernel's
// table work grows with B. Measured (us per call, up / down, LUT batch against matrix cores, medians of interleaved
// runs): 70B MLP layers B = 2 33.1 / 35.5 against 43.5 / 44.7, B = 4 41.0 / 42.2 against 43.3 / 44.1, B = 8 84.6 /
// 91.5 against 47.3 / 47.6; 7B MLP layers (fewer than four 1024-row units per CU, where the LUT batch kernel's
// 1024-row workgroups do not fill the chip) B = 2 14.8 / 17.7 against 13.8 / 14.9, B = 4 16.4 / 19.3 against 13.9 /
// 15.0. So mu = 8 uses the LUT batch kernel up to B = 4 on large layers and the matrix cores otherwise; mu = 4 (whose
// LUT path for B >= 2 is the generic kernel) always the matrix cores. The crossover, in 1024-row units U = ceil(M /
// 1024) x super-chunks, moves with B. At B = 2 the LUT batch kernel wins from U = 650 (us, matrix cores -> LUT batch:
// 10240x8192 with 2 bases + 1% (U = 650) 19.3 -> 17.3; with 3 bases + 5%: 7168x8192 (686) 20.2 -> 18.1, 8192x7168
// (688, row-complete matrix cores) 17.9 -> 17.1, 8192x8192 (784) 20.9 -> 19.9, 10240x8192 (980) 23.9 -> 19.6;
// 4096x11008 with 4 bases (688) 21.0 -> 19.2) and loses up to U = 540 (5120x13824 with 2 bases 18.3 -> 18.6, 8192x8192
// with 2 bases + 1% (520) 15.9 -> 16.9, 7B MLP (363, 352) 13.7 -> 14.5, 14.3 -> 16.8). At B = 3 and 4 it wins at U =
// 980 (24.0 -> 22.3, 24.2 -> 22.9) and loses at U = 784 and below (21.3 -> 22.1, 20.9 -> 22.3). Thresholds: U >= 2.25
// units per CU at B = 2, >= 3.5 at B = 3 and 4. FLUXBIN_MFMA=1 / 0 forces the choice (tests and measurements).
static bool use_mfma(const fluxbin_layer& L, int B, int cus, const fluxbin_tuning& tu) {
  const int forced = tu.mfma;
  if (forced == 0 || forced == 1) return forced == 1;
  const int quarters = B == 2 ? 9 : 14;   // LUT batch kernel from U >= quarters / 4 units per CU
  const bool small = 4 * ceil_div(L.shape.M, 1024) * L.NSC < int64_t(quarters) * cus;
  return L.shape.mu == 4 || B > 4 || small;
}

// Row-complete batch-1 kernel: coarse row scales, or 8 / 16 fine groups per salient chunk at mu = 8, x staged in LDS (N <= kRwMaxN), at most kRwSteps super-chunks
// per wavefront. Chosen for layers of at most one 16-row workgroup per CU with at most 64 super-chunks (four per
// wavefront of 16), or 128 on layers of at most a quarter of that. us per call, split-tile kernel -> row-complete
// kernel (16 wavefronts, graph-timed, medians of interleaved runs): 4096x4096 2b 7.63 -> 5.80, 4b 8.69 -> 8.26, 7B
// attention 4096x4096 (2+1, 2%) 8.26 -> 5.98, 2048x4096 7.79 -> 5.31, 3072x4096 3+1 (49 super-chunks) 8.40 -> 7.00,
// 1024x8192 2+1 (65) 8.36 -> 7.20, 1024x8192 3+1 (98) 9.35 -> 9.05; even or slower with more super-chunks per
// wavefront: 4096x11008 2b (86) 9.47 -> 9.68. FLUXBIN_ROWS=1 / 0 forces the choice where the layer allows it.
// *rb: rows per lane, 1 (16 rows per workgroup), 2 or 3 (32 or 48 rows; mu = 8).
static bool use_rows(const fluxbin_layer& L, const Derived& dv, int cus, const fluxbin_tuning& tu, int* rb) {
  const bool fine_ok = dv.Gcg == 1 && (dv.Gcs == 1 || (L.shape.mu == 8 && (dv.Gcs == 8 || dv.Gcs == 16)));
  *rb = 1;
  if (!fine_ok || L.shape.N > kRwMaxN || L.NSC > 8 * kRwSteps) return false;
  // its buffer loads take 32-bit offsets into the sign and row-scale sections
  if (dv.NCP * dv.Mp * 16 >= (int64_t(1) << 31) || dv.NRP * dv.Mp * 2 >= (int64_t(1) << 31)) return false;
  const bool rb2_ok = L.shape.mu == 8;   // with coarse row scales or 8 / 16 fine groups per salient chunk (fine_ok)
  if (tu.rows == 2 || tu.rows == 3) {
    *rb = tu.rows;
    return rb2_ok;
  }
  if (tu.rows == 0 || tu.rows == 1) return tu.rows == 1;
  const int64_t wgs = ceil_div(L.shape.M, 16);
  // up to one 16-row workgroup per CU: App. E.4 4096x11008 (86-97 super-chunks) 2b 10.1 -> 9.3, s8 11.6 -> 10.7, s16
  // 13.5 -> 11.2 us against the split-tile kernel; 4096x4096 8.2 -> 5.6
  if (wgs <= cus) return L.NSC <= 128;
  // Two rows per lane where 32-row workgroups fill the CUs once (more than half of them, at most one each) and each
  // workgroup's table work stays small: 8192 x 8192 with 2 bases + 1% (65 super-chunks, 256 workgroups) 12.2 -> 11.0
  // us against the split-tile kernel. With more workgroups than CUs the second workgroups on a CU double its time
  // (11008 rows: 344 workgroups, no faster), with fewer the idle CUs cost more than the reduction saved (4096 rows:
  // 5.7 -> 6.6 us), and 98 super-chunks (3 bases + 5%) were slower.
  const int64_t wgs32 = ceil_div(L.shape.M, 32);
  if (rb2_ok && 2 * wgs32 > cus && wgs32 <= cus && L.NSC <= 80) {
    *rb = 2;
    return true;
  }
  // three rows per lane (48-row workgroups) where 32-row ones would be more than the CUs, 48-row ones still keep
  // three quarters of them busy and the super-chunks are few: 11008x4096 (33 super-chunks) 9.5 -> 8.7 us; the fused
  // 10240x8192 q|k|v layer with 2 bases + 1% (65) was slower, 13.0 -> 13.9
  const int64_t wgs48 = ceil_div(L.shape.M, 48);
  if (rb2_ok && wgs32 > cus && wgs48 <= cus && 4 * wgs48 > 3 * cus && L.NSC <= 48) {
    *rb = 3;
    return true;
  }
  return false;
}

// Row-complete matrix-core kernel for B = 2..8 (16 or 32 rows per workgroup, every super-chunk of them, no split
// tiles): the first fitting shape of 16 wavefronts x 16 rows (one workgroup per CU), 8 wavefronts x 32 rows (two per
// CU), 16 wavefronts x 32 rows; fitting: the grid within one wave of workgroups, LDS (activation blocks of every
// column block, column-scale pairs of every chunk, sign scratch) within the CU's 160 KB, at most kMrSteps
// super-chunks per wavefront, buffer offsets below 2^31. By default only the first shape, on layers of half a
// workgroup to one workgroup per CU: 7B attention 4096x4096 at B = 2 / 4 / 8 11.1 / 11.3 / 11.6 -> 8.4 / 8.5 / 8.9 us
// (split-tile matrix-core kernel -> this); the 32-row shapes were slower than the split-tile kernel (7B gate/up
// 11008x4096 at B = 2: 13.2 -> 15.0 us: four to five units per wavefront, two in flight). FLUXBIN_MFMA_ROWS=0 never,
// 1 wherever it fits.
static bool use_mfma_rows(const fluxbin_layer& L, const Derived& dv, int B, int cus, const fluxbin_tuning& tu,
                          int* waves, int* rb) {
  if (tu.mfma_rows == 0 || tu.mfma == 0 || tu.generic) return false;
  if (tu.mfma_rows != 1 && !use_mfma(L, B, cus, tu)) return false;   // sizes where the LUT batch kernel is faster
  const int64_t wgs16 = ceil_div(L.shape.M, 16);
  // Taken where 16-row workgroups fill between half and all of the CUs, or where the shape's workgroups are at most
  // one per CU and the layer has at most 88 super-chunks (B = 2 / 4, µs against the split-tile matrix-core kernel:
  // 5120x5120 12.9 / 13.0 -> 10.1 / 10.2, 8192x8192 with 2 bases + 1% 16.8 / 17.2 -> 15.6 / 15.6, 1024x8192 11.8 /
  // 11.8 -> 10.4 / 10.4, 8192x7168 (86 super-chunks) 19.1 / 19.0 -> 17.8 / 17.9; with more workgroups than CUs (11008
  // rows: 344 of 32 rows) or 98 super-chunks it was slower)
  const bool fill = wgs16 <= cus && 2 * wgs16 >= cus;
  if (dv.NCP * dv.Mp * 16 >= (int64_t(1) << 31) || dv.NRP * dv.Mp * 2 >= (int64_t(1) << 31)) return false;
  const int bp = B <= 4 ? 4 : 8;
  const int64_t nblk = dv.ncg + (dv.NCP - L.shape.Kb * dv.ncg);
  const int64_t dyn = mfma_rows_lds_bytes(dv.NCP, nblk, bp);
  const int shapes[3][3] = {{16, 1, 1}, {8, 2, 2}, {16, 2, 1}};   // waves, row blocks, workgroups per CU
  for (const auto& sh : shapes) {
    const int64_t stat = int64_t(sh[0]) * sh[1] * 1024 + 2 * 2 * sh[0] * kMrSteps * 4;
    const int64_t wgs = ceil_div(L.shape.M, 16 * sh[1]);
    if (L.NSC <= int64_t(sh[0]) * kMrSteps && (stat + dyn) * sh[2] <= 160 * 1024 && wgs <= int64_t(cus) * sh[2] &&
        (tu.mfma_rows == 1 || fill || (wgs <= cus && L.NSC <= 88))) {
      *waves = sh[0];
      *rb = sh[1];
      return true;
    }
  }
  return false;
}

static uint64_t layer_counter_bytes(int64_t M) {
  return round_up256(uint64_t(ceil_div(M, 256) + 4) * uint64_t(kCounterStride) * 4u);
}

// Rows of a full batch tile (calls with more batch rows run as several launches): 32 on layers the matrix-core kernel
// takes (one row scale per chunk), whose sign decode then serves two 16-row MFMA tiles, else 16. Layers with 8 or 16
// fine salient row-scale groups at mu = 8 (the paper's s16 / s8 configurations), which only the generic kernel takes at
// B >= 2, run B <= 8 rows as B launches of the batch-1 kernels instead: faster on all eight App. E.4 s8 / s16 layers
// at B = 2, 4 and 8 (us per call, generic kernel -> per-row batch-1 launches: 4096x4096 s8 B = 2 15.1 -> 12.1, B = 8
// 59.5 -> 46.4; 5120x13824 s8 B = 2 55.7 -> 30.1, B = 8 139.5 -> 115.3). FLUXBIN_BATCH_TILE=16 keeps 16-row tiles.
static int batch_tile_rows(const fluxbin_layer& L, const fluxbin_tuning& tu, int B) {
  const Derived dv = derive(L.shape);
  if (!tu.generic && tu.batch_tile != kMaxBatch && B <= 8 && L.shape.mu == 8 && dv.Gcg == 1 &&
      (dv.Gcs == 8 || dv.Gcs == 16))
    return 1;
  if (tu.generic || dv.Gcg > 1 || dv.Gcs > 1 || tu.mfma == 0 || tu.mfma_depth == 3 || tu.mfma_r2 == 0 ||
      tu.batch_tile == kMaxBatch)
    return kMaxBatch;
  return kMaxBatchMfma;
}

fluxbin_status make_plan(const fluxbin_layer& L, int B, Plan* p, bool allow_rows) {
  const int cus = device_cu_count();
  if (cus <= 0) return fail(FLUXBIN_ERR_HIP, "cannot query the current HIP device");
  std::memset(p, 0, sizeof(*p));
  const fluxbin_tuning tu = tuning_snapshot();
  if (B < 1 || (B > kMaxBatch && batch_tile_rows(L, tu, B) < B))
    return fail(FLUXBIN_ERR_UNSUPPORTED, "no launch plan for %d batch rows in one launch on this layer", B);
  const int force_generic = tu.generic;
  const int rpt_env = tu.rpt;
  int per_cu = tu.blocks_per_cu;
  // Fine row-scale groups (groups shorter than a chunk): the batch-1 kernel's instances for them take mu = 8 layers
  // whose fine groups are on the salient side only (the paper's s8/s16 configurations), one unit ahead, 512 or 1024
  // threads; every other case with fine groups runs the generic kernel (the matrix-core and LUT batch kernels apply one
  // row scale per chunk).
  const Derived dv = derive(L.shape);
  const bool fine = dv.Gcg > 1 || dv.Gcs > 1;
  // the batch-1 instances for fine groups: salient side only, 8 or 16 groups per chunk (s = 16 or 8 at mu = 8)
  const bool b1_fine_ok = L.shape.mu == 8 && dv.Gcg == 1 && (dv.Gcs == 8 || dv.Gcs == 16);
  p->nt = 256;
  int rw_rb = 1;
  if (B == 1 && !force_generic && allow_rows && use_rows(L, dv, cus, tu, &rw_rb)) {
    // row-complete batch-1 kernel: 16 rows per workgroup (32 with two rows per lane), every super-chunk of them, no
    // cross-workgroup reduction; 16 wavefronts, two units requested ahead (4 and 8 wavefronts, and 4 or 6 units ahead,
    // measured slower or equal)
    p->kernel = 4;
    p->nt = rw_rb == 2 ? 1024 : ((tu.nt == 256 && L.NSC <= 4 * kRwSteps) ? 256 : (tu.nt == 512 ? 512 : 1024));
    p->rpt = 1;
    p->rows = 16 * rw_rb;
    p->depth = rw_rb == 2 ? 2 : ((tu.depth == 4 || tu.depth == 6) ? tu.depth : 2);
    p->bg = 1;
    p->n_groups = 1;
    p->bpad = 1;
    p->n_tiles = ceil_div(L.shape.M, p->rows);
    p->units = p->n_tiles * L.NSC;
    p->blocks = p->n_tiles;
    p->ws_counters_off = 0;
    p->ws_partials_off = layer_counter_bytes(L.shape.M);
    p->ws_bytes = p->ws_partials_off;   // no workspace of its own: the counter region every plan of the layer keeps
    return FLUXBIN_OK;
  }
  int mr_waves = 0, mr_rb = 0;
  if (B >= 2 && B <= 8 && !force_generic && !fine && use_mfma_rows(L, dv, B, cus, tu, &mr_waves, &mr_rb)) {
    // row-complete matrix-core kernel: no split tiles, no second kernel, activations staged once per workgroup
    p->kernel = 5;
    p->nt = 64 * mr_waves;
    p->rpt = 1;
    p->rows = 16 * mr_rb;
    p->depth = 2;
    p->bg = B <= 4 ? 4 : 8;
    p->n_groups = 1;
    p->bpad = p->bg;
    p->n_tiles = ceil_div(L.shape.M, p->rows);
    p->units = p->n_tiles * L.NSC;
    p->blocks = p->n_tiles;
    p->ws_counters_off = 0;
    p->ws_partials_off = layer_counter_bytes(L.shape.M);
    p->ws_image_off = p->ws_partials_off;   // no partial sums: the staging image follows the counter region
    p->ws_bytes = p->ws_image_off +
                  uint64_t(mfma_rows_image_dwords(dv.NCP, dv.ncg + (dv.NCP - L.shape.Kb * dv.ncg), p->bpad)) * 4u;
    return FLUXBIN_OK;
  }
  if (B == 1 && !force_generic && (!fine || b1_fine_ok)) {   // batch-1 kernel (mu = 8 or 4)
    p->kernel = 0;
    const int nt_env = tu.nt;
    // units of sign data requested ahead of the one being looked up: one (two units, 64 KB per CU, in flight) already
    // keeps HBM saturated; deeper rings only add queueing and prologue latency
    const int depth_env = tu.depth;
    p->depth = (depth_env == 2 || depth_env == 3) ? depth_env : 1;
    // layers whose sign stream is small for the chip overlap the activation and sign round trips (see the kernel)
    const int early_env = tu.early;
    const int64_t sign_bytes = int64_t(L.NSC) * 2 * L.Mp * 16;
    p->early = early_env >= 0 ? early_env != 0 : sign_bytes <= (int64_t(32) << 20);
    // mu = 8: 1024-thread workgroups, one per CU, amortize each table over the most rows and keep the fewest,
    // longest pipelines, which pays once a layer has at least four 1024-row units per CU (the 70B MLP layers: 0.5 us
    // faster than 512 threads). Below that, 512-thread workgroups (up to two per CU) keep more CUs busy: measured
    // 11008x4096 10.2 -> 8.7 us (121 -> 242 workgroups of three units), 4096x11008 10.9 -> 9.4, 8192x8192 with two
    // bases 11.5 -> 11.1, 10240x8192 with three bases 13.6 -> 13.1; 256 threads were slower on every layer measured
    // (1024x8192: 9.8 us against 8.4 at 512).
    // mu = 4 does twice the lookups per row and column of mu = 8; there two 512-thread workgroups per CU, each
    // covering the other's barriers, measured 2 to 2.5 us faster than one 1024-thread workgroup on the 8192- and
    // 28672-row MLP layers: 512 threads at most, fewer for layers with fewer than one unit per CU.
    if (nt_env == 256 || nt_env == 512 || nt_env == 1024) {
      p->nt = nt_env;
      if (fine && p->nt == 256) p->nt = 512;
    } else if (L.shape.mu == 8) {
      p->nt = ceil_div(L.shape.M, 1024) * L.NSC >= 4 * int64_t(cus) ? 1024 : 512;
    } else {
      p->nt = 512;
      while (p->nt > 256 && ceil_div(L.shape.M, p->nt) * L.NSC < cus) p->nt /= 2;
    }
    if (fine) p->depth = 1;
    if (per_cu < 1 || per_cu > 8) per_cu = 1024 / p->nt;
    p->bg = 1;
    p->n_groups = 1;
  } else if (B >= 2 && !force_generic && !fine && use_mfma(L, B, cus, tu)) {
    // small batch on the matrix cores: the sign decode per bit is shared by all batch rows (B <= 16 fit one MFMA tile)
    p->kernel = 3;
    p->nt = 256;
    p->rpt = 1;   // four 16-row blocks per wavefront: 256-row tiles
    // units of data requested ahead: two (measured 2-8 us faster than three on the 70B MLP layers at B = 2..16)
    const int depth_env = tu.mfma_depth;
    p->depth = depth_env == 3 ? 3 : 2;
    p->bg = B <= 4 ? 4 : (B <= 8 ? 8 : (B <= 16 ? 16 : 32));
    p->n_groups = 1;
    // split tiles reduced by a second kernel (FLUXBIN_MFMA_R2=0: by the tile counters, as at batch 1): measured
    // on the 70B MLP layers, up / down, 58.6 / 78.7 -> 57.2 / 59.3 us at B = 16, 48.0 / 57.7 -> 46.5 / 47.1 at B = 8,
    // 45.5 / 48.8 -> 42.6 / 43.6 at B = 4; 7B MLP layers 18.8 / 19.0 -> 15.1 / 17.1 at B = 4
    p->reduce2 = p->depth == 2 && tu.mfma_r2 != 0;
    // three 256-thread workgroups per CU (the kernel's occupancy at 16 and 32 batch rows; three units ahead, or four
    // workgroups per CU at 16 rows: no faster)
    if (per_cu < 1 || per_cu > 8) per_cu = 3;
    if (p->bg == 32 && !p->reduce2)
      return fail(FLUXBIN_ERR_UNSUPPORTED, "32-row matrix-core launches need the second-kernel reduction");
  } else if (L.shape.mu == 8 && B >= 2 && !force_generic && !fine) {
    // small batch: 1024-row tiles, one super-chunk per unit (the batch-1 sign stream), batch in groups of four rows
    // (two for B = 2: half the table entries and lookup additions of a padded group of four)
    p->kernel = 2;
    p->nt = 1024;
    const int depth_env = tu.depth;
    p->depth = (depth_env == 2 || depth_env == 3) ? depth_env : 1;
    p->bg = B == 2 ? 2 : 4;
    p->n_groups = int(ceil_div(B, 4));   // every group holds at least one batch row (the grid's y extent)
    // one batch group: split tiles reduced by a second kernel (FLUXBIN_BAT_R2=0: by the tile counters). Measured on the
    // 70B MLP layers, up / down: B = 2 37.6 / 40.6 -> 33.8 / 35.0 us, B = 4 46.0 / 50.2 -> 40.3 / 41.7 us
    p->reduce2 = p->n_groups == 1 && p->depth == 1 && tu.bat_r2 != 0;
    if (per_cu < 1 || per_cu > 8) per_cu = 1;
  } else {
    p->kernel = 1;
    p->bg = B == 1 ? 1 : (B == 2 ? 2 : 4);
    p->n_groups = int((B + p->bg - 1) / p->bg);
    if (p->n_groups == 3) p->n_groups = 4;  // instantiated batch paddings: 1, 2, 4, 8, 16
    if (per_cu < 1 || per_cu > 8) per_cu = 2;
  }
  if (B > kMaxBatch && p->kernel != 3)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "%d batch rows in one launch need the matrix-core kernel", B);
  const int blocks_env = tu.blocks;   // tuning override: grid size target
  const int64_t target = blocks_env > 0 ? blocks_env : int64_t(cus) * per_cu;
  p->bpad = p->bg * p->n_groups;
  const int64_t steps = p->kernel == 1 ? (2 * L.NSC) * p->n_groups : L.NSC;
  // instantiated rows per thread: batch-1 kernel 4/2/1 at 256 threads, 2/1 at 512 and 1024 (default 1: one row per
  // thread gives the most units to balance and the lightest registers); the generic kernel 4 only for mu = 8 with
  // <= 2 batch rows
  int rpt_max = (p->kernel == 0 || (L.shape.mu == 8 && p->bpad <= 2)) ? 4 : 2;
  if (p->kernel == 0) rpt_max = p->nt == 256 ? 4 : 2;
  int chosen = 1;
  if (p->kernel == 3) {
    chosen = p->rpt;
  } else if (p->kernel != 1) {
    chosen = 1;   // the batch-1 and small-batch kernels: one row per thread
  } else if (rpt_env == 1 || rpt_env == 2 || rpt_env == 4) {
    chosen = rpt_env > rpt_max ? rpt_max : rpt_env;
  } else if (p->kernel == 0) {
    chosen = 1;
  } else {
    for (int rpt = rpt_max; rpt >= 1; rpt /= 2) {
      const int64_t tiles = ceil_div(L.shape.M, int64_t(p->nt) * rpt);
      if (tiles * steps >= 2 * target || rpt == 1) {
        chosen = rpt;
        break;
      }
    }
  }
  p->rpt = chosen;
  p->rows = p->nt * p->rpt;
  p->n_tiles = ceil_div(L.shape.M, p->rows);
  p->units = p->n_tiles * steps;
  if (p->units > (int64_t(1) << 30))
    return fail(FLUXBIN_ERR_UNSUPPORTED, "layer too large for one launch (%lld work units)", (long long)p->units);
  p->blocks = p->units < target ? p->units : target;
  // small layers: give every workgroup at least a few units, so that its fixed start-up cost is amortized and a split
  // tile has fewer contributors to reduce. Three, or two where workgroups of two units still number at most one per
  // CU (4096x4096: 8.2 -> 8.0 us at mu = 8, 8.5 -> 8.2 us at mu = 4; 1024x8192: 8.6 -> 8.4 us; with more workgroups
  // than CUs some CUs would run two of them: 11008x4096 8.7 -> 9.9 us).
  const int min_units_dflt = ceil_div(p->units, 2) <= cus ? 2 : 3;
  const int min_units = tu.min_units >= 0 ? tu.min_units : min_units_dflt;
  if (min_units > 1 && p->kernel == 0 && p->blocks > 1 && ceil_div(p->units, p->blocks) < min_units)
    p->blocks = ceil_div(p->units, int64_t(min_units)) > 0 ? ceil_div(p->units, int64_t(min_units)) : 1;
  // The batch-1 kernel stages the folded activations of all its units at once: at most b1_max_units(nt) per
  // workgroup. 1024-thread mu = 8 plans whose units need 17..24 per workgroup to fit one wave of workgroups (the fused
  // 57344x8192 gate|up layer with 3 bases: 5488 units, 21.4 per workgroup) take the instance that stages up to
  // kBigUnits, one wave instead of two: 41.9 -> 39.3 us. FLUXBIN_BIG_UNITS=0 keeps them at 16 units.
  p->xv = 0;
  if (p->kernel == 0 && p->nt == 1024 && L.shape.mu == 8 && !fine && p->depth == 1 && !p->early && tu.big_units != 0 &&
      blocks_env <= 0 && ceil_div(p->units, p->blocks) > b1_max_units(1024) &&
      ceil_div(p->units, int64_t(cus) * per_cu) <= kBigUnits)
    p->xv = kBigUnits;
  const int64_t b1_cap = p->xv ? p->xv : b1_max_units(p->nt);
  if (p->kernel == 0 && ceil_div(p->units, p->blocks) > b1_cap) p->blocks = ceil_div(p->units, b1_cap);
  // The same for the LUT batch kernel with the second-kernel reduction (one batch group, one unit ahead): up to
  // kBigUnits instead of kBatMaxUnits where that fits the layer into one wave (fused gate|up, 4-base layers).
  if (p->kernel == 2 && p->reduce2 && p->n_groups == 1 && p->depth == 1 && tu.big_units != 0 && blocks_env <= 0 &&
      ceil_div(p->units, p->blocks) > kBatMaxUnits && ceil_div(p->units, int64_t(cus) * per_cu) <= kBigUnits)
    p->xv = kBigUnits;
  const int64_t bat_cap = p->kernel == 2 && p->xv ? p->xv : kBatMaxUnits;
  if (p->kernel == 2 && ceil_div(p->units, p->blocks) > bat_cap) p->blocks = ceil_div(p->units, bat_cap);
  // the matrix-core kernel: at least three units per workgroup (fewer split tiles to reduce, each workgroup's start-up
  // amortized), as long as that leaves a workgroup for every CU. 7B MLP layers (about 1400 units), us per call up / down
  // at 768 -> 512 -> 256 workgroups: B = 8 17.0 / 19.5 -> 14.7 / 16.7 -> 16.4 / 16.6, B = 16 22.6 / 24.7 -> 17.9 /
  // 19.9 -> 18.8 / 18.8.
  if (p->kernel == 3 && blocks_env <= 0 && ceil_div(p->units, p->blocks) < 3) {
    const int64_t floor_blocks = p->units < cus ? p->units : int64_t(cus);
    const int64_t b3 = ceil_div(p->units, 3);
    p->blocks = b3 > floor_blocks ? b3 : floor_blocks;
  }
  if (p->kernel == 3 && ceil_div(p->units, p->blocks) > kMfMaxUnits) p->blocks = ceil_div(p->units, kMfMaxUnits);
  // More workgroups than the chip holds at once (the caps above on large layers): whole waves of workgroups, each with
  // fewer units, instead of one full wave and a small second one that leaves most CUs idle (57344x8192 with 2 bases at
  // B = 4: 304 one-per-CU workgroups of 12 units -> 512 of 7.1).
  const int64_t resident = int64_t(cus) * per_cu;
  if (p->kernel != 1 && blocks_env <= 0 && p->blocks > resident) {
    const int64_t whole = ceil_div(p->blocks, resident) * resident;
    p->blocks = whole < p->units ? whole : p->units;
  }
  // Unit ranges aligned to tiles (kpt workgroups per tile, each a contiguous part of one tile) for the split-tile
  // kernels, where that fits one wave of resident workgroups: about as many workgroups as the balanced split, and at
  // most its most units per workgroup. A balanced range over a tile boundary ends two tiles (two transposes or stores
  // of partial sums, two counter bumps), and such workgroups end last; an aligned range ends one. Matrix-core kernel,
  // 70B MLP down projection (32 tiles of 342 units, 768 workgroups): 49.7 -> 45.6 us at B = 8, 73.9 -> 70.3 at B = 32;
  // 7B MLP (43 and 16 tiles, about 470 workgroups) 2 to 8 % faster at B = 8..32. The 70B up projection's 112 tiles of
  // 98 units need 7 per tile, 784 workgroups: one wave of 768 and a tail, so the matrix-core kernel keeps the balanced
  // split there. FLUXBIN_ALIGN=0 keeps the balanced split everywhere; k > 0 forces k per tile.
  p->kpt = 0;
  if ((p->kernel == 0 || p->kernel == 2 || p->kernel == 3) && tu.align != 0 && blocks_env <= 0 && p->n_tiles > 0) {
    const int64_t steps = p->units / p->n_tiles;
    const int64_t cap = p->kernel == 0 ? b1_cap : (p->kernel == 2 ? bat_cap : kMfMaxUnits);
    const int64_t k_round = (p->blocks + p->n_tiles / 2) / p->n_tiles;
    const int64_t k_units = ceil_div(steps, ceil_div(p->units, p->blocks));
    int64_t kpt = tu.align > 0 ? tu.align : (k_round > k_units ? k_round : k_units);
    const int64_t kmin = ceil_div(steps, cap);
    if (kpt < kmin) kpt = kmin;
    if (kpt > steps) kpt = steps;
    // batch-1 kernel with more workgroups than CUs and at most three units each: the tiles' parts one unit longer
    // than the rest then share CUs (App. E.4 5120x13824: 10 tiles of 51 parts, 13.0 / 15.2 / 14.4 us balanced against
    // 13.9 / 16.0 / 15.3 aligned for 2b / s8 / s16), so the balanced split stays
    const bool short_parts = p->kernel == 0 && p->n_tiles * kpt > cus && ceil_div(steps, kpt) <= 3;
    if (tu.align > 0 || (p->n_tiles * kpt <= resident && !short_parts)) {
      p->kpt = int(kpt);
      p->blocks = p->n_tiles * kpt;
    }
  }
  p->ws_counters_off = 0;
  // the small-batch kernel runs one row of workgroups per group of four batch rows, each with its own counters
  const uint64_t counter_sets = p->kernel == 2 ? uint64_t(p->n_groups) : 1u;
  const uint64_t counter_bytes = counter_sets * round_up256(uint64_t(p->n_tiles) * uint64_t(kCounterStride) * 4u);
  // The counter region is the same for every launch plan of the layer: room for ceil(M/256) + 4 tile counters (the
  // most any plan uses: 256-row tiles, or four sets of 1024-row tiles). So no plan's partial sums overlap another
  // plan's counters, and calls of one layer with any batch size can share a workspace.
  p->ws_partials_off = layer_counter_bytes(L.shape.M);
  if (counter_bytes > p->ws_partials_off)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "launch plan needs %llu bytes of tile counters, the layer's region holds %llu",
                (unsigned long long)counter_bytes, (unsigned long long)p->ws_partials_off);
  p->ws_bytes = p->ws_partials_off + uint64_t(p->blocks) * 2u * uint64_t(p->rows) * uint64_t(p->bpad) * 4u;
  if (p->kernel == 3 && p->bpad > 8) {   // the activation images of every super-chunk, written by a first kernel
    p->ws_image_off = round_up256(p->ws_bytes);
    p->ws_bytes = p->ws_image_off + uint64_t(L.NSC) * uint64_t(mf_image_dwords(p->bpad)) * 4u;
  }
  return FLUXBIN_OK;
}

static bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + nb && pb < pa + na;
}

// Copies an array to a fresh device allocation (host-input packing path).
static fluxbin_status stage(const void* h, size_t bytes, void** d, std::vector<void*>& owned) {
  *d = nullptr;
  if (!h || bytes == 0) return FLUXBIN_OK;
  hipError_t e = hipMalloc(d, bytes);
  if (e != hipSuccess) return hip_fail(e, "hipMalloc (pack staging)");
  owned.push_back(*d);
  e = hipMemcpy(*d, h, bytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy (pack staging)");
  return FLUXBIN_OK;
}

}  // namespace fluxbin

using namespace fluxbin;

extern "C" {

const char* fluxbin_status_string(fluxbin_status s) {
  // C callers may pass any int; read it as one (in C++ a value outside the enumerators' range is not a valid
  // fluxbin_status, and switching on it directly is undefined)
  int v;
  std::memcpy(&v, &s, sizeof(v));
  switch (v) {
    case FLUXBIN_OK: return "ok";
    case FLUXBIN_ERR_INVALID_ARG: return "invalid argument";
    case FLUXBIN_ERR_UNSUPPORTED: return "unsupported";
    case FLUXBIN_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case FLUXBIN_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* fluxbin_last_error_message(void) { return g_msg; }

fluxbin_status fluxbin_pack_query(const fluxbin_shape* shape, size_t* packed_bytes) {
  g_msg[0] = 0;
  fluxbin_status st = check_shape(shape);
  if (st != FLUXBIN_OK) return st;
  if (!packed_bytes) return fail(FLUXBIN_ERR_INVALID_ARG, "packed_bytes is NULL");
  *packed_bytes = static_cast<size_t>(offsets(*shape, derive(*shape)).total);
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_pack(const fluxbin_shape* shape, const fluxbin_weights* w, void* d_packed, size_t packed_bytes,
                            fluxbin_layer* out, hipStream_t stream) {
  g_msg[0] = 0;
  fluxbin_status st = check_shape(shape);
  if (st != FLUXBIN_OK) return st;
  if (!w) return fail(FLUXBIN_ERR_INVALID_ARG, "weights is NULL");
  if (!out) return fail(FLUXBIN_ERR_INVALID_ARG, "out is NULL");
  if (!d_packed) return fail(FLUXBIN_ERR_INVALID_ARG, "d_packed is NULL");
  const fluxbin_shape& s = *shape;
  const Derived d = derive(s);
  const Offsets o = offsets(s, d);
  if (packed_bytes < o.total)
    return fail(FLUXBIN_ERR_BUFFER_TOO_SMALL, "packed buffer has %zu bytes, needs %llu", packed_bytes,
                (unsigned long long)o.total);
  if (!w->signs || !w->alpha_r || !w->alpha_c) return fail(FLUXBIN_ERR_INVALID_ARG, "global weight pointer is NULL");
  const bool sal = s.S > 0 && s.Ks > 0;
  if (s.S > 0 && !w->sal_idx) return fail(FLUXBIN_ERR_INVALID_ARG, "sal_idx is NULL with S > 0");
  if (sal && (!w->sal_signs || !w->alpha_sr || !w->alpha_sc))
    return fail(FLUXBIN_ERR_INVALID_ARG, "salient weight pointer is NULL with S > 0 and Ks > 0");
  if (w->inputs_on_device != 0 && w->inputs_on_device != 1)
    return fail(FLUXBIN_ERR_INVALID_ARG, "inputs_on_device must be 0 or 1");

  const int64_t W = ceil_div(s.N, 32);
  const size_t n_signs = size_t(s.Kb) * s.M * W * 4;
  const size_t n_ar = size_t(s.Kb) * s.M * d.Gr * 2;
  const size_t n_ac = size_t(s.Kb) * s.N * 2;
  const size_t n_idx = size_t(s.S) * 4;
  const size_t n_ss = sal ? size_t(s.Ks) * s.M * W * 4 : 0;
  const size_t n_asr = sal ? size_t(s.Ks) * s.M * d.Gs * 2 : 0;
  const size_t n_asc = sal ? size_t(s.Ks) * s.N * 2 : 0;

  // The salient set must be strictly increasing and in range: checked on the host before any kernel reads it.
  std::vector<int32_t> idx(size_t(s.S));
  if (s.S > 0) {
    if (w->inputs_on_device) {
      hipError_t e = hipMemcpyAsync(idx.data(), w->sal_idx, n_idx, hipMemcpyDeviceToHost, stream);
      if (e == hipSuccess) e = hipStreamSynchronize(stream);
      if (e != hipSuccess) return hip_fail(e, "copying sal_idx to the host");
    } else {
      std::memcpy(idx.data(), w->sal_idx, n_idx);
    }
    for (int64_t t = 0; t < s.S; ++t) {
      if (idx[t] < 0 || idx[t] >= s.N)
        return fail(FLUXBIN_ERR_INVALID_ARG, "sal_idx[%lld] = %d out of range [0, N)", (long long)t, idx[t]);
      if (t > 0 && idx[t] <= idx[t - 1])
        return fail(FLUXBIN_ERR_INVALID_ARG, "sal_idx is not strictly increasing at %lld", (long long)t);
    }
  }

  fluxbin_layer L;
  fill_layer(s, d_packed, packed_bytes, &L);

  if (w->inputs_on_device) {
    st = launch_pack(L, *w, w->sal_idx, stream);
    if (st != FLUXBIN_OK) return st;
  } else {
    std::vector<void*> owned;
    fluxbin_weights dw = *w;
    void* p = nullptr;
    auto release = [&]() {
      for (void* q : owned) (void)hipFree(q);
    };
    st = stage(w->signs, n_signs, &p, owned); dw.signs = (const uint32_t*)p;
    if (st == FLUXBIN_OK) { st = stage(w->alpha_r, n_ar, &p, owned); dw.alpha_r = (const uint16_t*)p; }
    if (st == FLUXBIN_OK) { st = stage(w->alpha_c, n_ac, &p, owned); dw.alpha_c = (const uint16_t*)p; }
    if (st == FLUXBIN_OK) { st = stage(w->sal_idx, n_idx, &p, owned); dw.sal_idx = (const int32_t*)p; }
    if (st == FLUXBIN_OK && sal) { st = stage(w->sal_signs, n_ss, &p, owned); dw.sal_signs = (const uint32_t*)p; }
    if (st == FLUXBIN_OK && sal) { st = stage(w->alpha_sr, n_asr, &p, owned); dw.alpha_sr = (const uint16_t*)p; }
    if (st == FLUXBIN_OK && sal) { st = stage(w->alpha_sc, n_asc, &p, owned); dw.alpha_sc = (const uint16_t*)p; }
    dw.inputs_on_device = 1;
    if (st == FLUXBIN_OK) st = launch_pack(L, dw, dw.sal_idx, stream);
    if (st == FLUXBIN_OK) {
      hipError_t e = hipStreamSynchronize(stream);
      if (e != hipSuccess) st = hip_fail(e, "hipStreamSynchronize (pack)");
    } else {
      (void)hipStreamSynchronize(stream);
    }
    release();
    if (st != FLUXBIN_OK) return st;
  }
  *out = L;
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_layer_from_header(const void* header_host, void* d_packed, size_t packed_bytes,
                                         fluxbin_layer* out) {
  g_msg[0] = 0;
  if (!header_host || !d_packed || !out) return fail(FLUXBIN_ERR_INVALID_ARG, "NULL argument");
  Header h;
  std::memcpy(&h, header_host, sizeof(h));
  if (h.magic != kMagic) return fail(FLUXBIN_ERR_INVALID_ARG, "bad magic 0x%08x", h.magic);
  if (h.version != FLUXBIN_FORMAT_VERSION) return fail(FLUXBIN_ERR_UNSUPPORTED, "format version %u", h.version);
  fluxbin_status st = check_shape(&h.shape);
  if (st != FLUXBIN_OK) return st;
  const Derived d = derive(h.shape);
  const Offsets o = offsets(h.shape, d);
  if (h.total != o.total || h.off_signs != o.signs || h.NSC != d.NSC || h.Mp != d.Mp)
    return fail(FLUXBIN_ERR_INVALID_ARG, "header sizes are inconsistent with its shape");
  if (packed_bytes < o.total) return fail(FLUXBIN_ERR_BUFFER_TOO_SMALL, "packed buffer is too small");
  fill_layer(h.shape, d_packed, packed_bytes, out);
  return FLUXBIN_OK;
}

}  // extern "C"

// Batches larger than one launch's rows (batch_tile_rows: 16 or 32) run as consecutive launches of full batch tiles
// (the last one with the remaining rows), each with its own launch plan, one after another on the caller's stream and
// sharing the workspace (every launch leaves its counters at zero). Each tile reads the packed weights again: the batch
// dimension is tiled with a fixed per-launch on-chip footprint.
struct BatchTiles {
  Plan full, tail;     // plans of a full tile and of the last tile (tail rows < tile; unused if 0)
  int tile, n_full, tail_rows;
  uint64_t ws_bytes;   // the larger of the two plans' workspaces
};

static fluxbin_status batch_tiles(const fluxbin_layer& L, int B, int tile, BatchTiles* bt) {
  std::memset(bt, 0, sizeof(*bt));
  bt->tile = tile;
  bt->n_full = B / tile;
  bt->tail_rows = B % tile;
  if (bt->n_full > 0) {
    const fluxbin_status st = make_plan(L, tile, &bt->full);
    if (st != FLUXBIN_OK) return st;
    bt->ws_bytes = bt->full.ws_bytes;
  }
  if (bt->tail_rows > 0) {
    const fluxbin_status st = make_plan(L, bt->tail_rows, &bt->tail);
    if (st != FLUXBIN_OK) return st;
    if (bt->tail.ws_bytes > bt->ws_bytes) bt->ws_bytes = bt->tail.ws_bytes;
  }
  return FLUXBIN_OK;
}

extern "C" {

fluxbin_status fluxbin_workspace_query(const fluxbin_layer* layer, int32_t B, size_t* bytes) {
  g_msg[0] = 0;
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  if (!bytes) return fail(FLUXBIN_ERR_INVALID_ARG, "bytes is NULL");
  if (B < 1 || B > kMaxBatchCall) return fail(FLUXBIN_ERR_INVALID_ARG, "B = %d out of range [1, %d]", B, kMaxBatchCall);
  BatchTiles bt;
  st = batch_tiles(*layer, B, batch_tile_rows(*layer, tuning_snapshot(), B), &bt);
  if (st != FLUXBIN_OK) return st;
  *bytes = static_cast<size_t>(bt.ws_bytes);
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_workspace_init(void* d_workspace, size_t bytes, hipStream_t stream) {
  g_msg[0] = 0;
  if (!d_workspace && bytes) return fail(FLUXBIN_ERR_INVALID_ARG, "workspace is NULL");
  if (bytes % 4) return fail(FLUXBIN_ERR_INVALID_ARG, "workspace size must be a multiple of 4");
  if (bytes == 0) return FLUXBIN_OK;
  return launch_fill_zero(d_workspace, bytes, stream);
}

static fluxbin_status gemm_common(const fluxbin_layer* layer, int32_t B, const uint16_t* d_x, int64_t ldx, void* d_y,
                                  int64_t ldy, int32_t y_is_fp32, void* d_ws, size_t ws_bytes, hipStream_t stream) {
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  const fluxbin_shape& s = layer->shape;
  if (B < 1 || B > kMaxBatchCall) return fail(FLUXBIN_ERR_INVALID_ARG, "B = %d out of range [1, %d]", B, kMaxBatchCall);
  if (!d_x || !d_y) return fail(FLUXBIN_ERR_INVALID_ARG, "x or y is NULL");
  if (y_is_fp32 != 0 && y_is_fp32 != 1) return fail(FLUXBIN_ERR_INVALID_ARG, "y_is_fp32 must be 0 or 1");
  if (ldx < s.N) return fail(FLUXBIN_ERR_INVALID_ARG, "ldx = %lld < N", (long long)ldx);
  if (ldy < s.M) return fail(FLUXBIN_ERR_INVALID_ARG, "ldy = %lld < M", (long long)ldy);
  const size_t xb = (size_t(B - 1) * ldx + s.N) * 2;
  const size_t yb = (size_t(B - 1) * ldy + s.M) * (y_is_fp32 ? 4 : 2);
  if (ranges_overlap(d_x, xb, d_y, yb)) return fail(FLUXBIN_ERR_INVALID_ARG, "x and y overlap");
  BatchTiles bt;
  st = batch_tiles(*layer, B, batch_tile_rows(*layer, tuning_snapshot(), B), &bt);
  if (st != FLUXBIN_OK) return st;
  if (!d_ws) return fail(FLUXBIN_ERR_INVALID_ARG, "workspace is NULL");
  if (ws_bytes < bt.ws_bytes)
    return fail(FLUXBIN_ERR_BUFFER_TOO_SMALL, "workspace has %zu bytes, needs %llu", ws_bytes,
                (unsigned long long)bt.ws_bytes);
  if (ranges_overlap(d_ws, ws_bytes, d_y, yb) || ranges_overlap(d_ws, ws_bytes, d_x, xb))
    return fail(FLUXBIN_ERR_INVALID_ARG, "workspace overlaps x or y");
  const size_t y_elt = y_is_fp32 ? 4 : 2;
  for (int t = 0; t <= bt.n_full; ++t) {
    const int rows = t < bt.n_full ? bt.tile : bt.tail_rows;
    if (rows == 0) break;
    const int64_t b0 = int64_t(t) * bt.tile;
    st = launch_gemm(*layer, t < bt.n_full ? bt.full : bt.tail, rows, d_x + b0 * ldx, ldx,
                     static_cast<uint8_t*>(d_y) + size_t(b0) * size_t(ldy) * y_elt, ldy, y_is_fp32, d_ws, stream);
    if (st != FLUXBIN_OK) return st;
  }
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_lut_gemv(const fluxbin_layer* layer, const uint16_t* d_x, void* d_y, int32_t y_is_fp32,
                                void* d_workspace, size_t workspace_bytes, hipStream_t stream) {
  g_msg[0] = 0;
  const int64_t M = layer ? layer->shape.M : 0;
  const int64_t N = layer ? layer->shape.N : 0;
  return gemm_common(layer, 1, d_x, N, d_y, M, y_is_fp32, d_workspace, workspace_bytes, stream);
}

fluxbin_status fluxbin_lut_gemm_smallbatch(const fluxbin_layer* layer, int32_t B, const uint16_t* d_x, int64_t ldx,
                                           void* d_y, int64_t ldy, int32_t y_is_fp32, void* d_workspace,
                                           size_t workspace_bytes, hipStream_t stream) {
  g_msg[0] = 0;
  return gemm_common(layer, B, d_x, ldx, d_y, ldy, y_is_fp32, d_workspace, workspace_bytes, stream);
}

fluxbin_status fluxbin_lut_gemv_noalloc(const fluxbin_layer* layer, const uint16_t* d_x, void* d_y, int32_t y_is_fp32,
                                        hipStream_t stream) {
  g_msg[0] = 0;
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  if (!d_x || !d_y) return fail(FLUXBIN_ERR_INVALID_ARG, "x or y is NULL");
  if (y_is_fp32 != 0 && y_is_fp32 != 1) return fail(FLUXBIN_ERR_INVALID_ARG, "y_is_fp32 must be 0 or 1");
  const size_t xb = size_t(layer->shape.N) * 2;
  const size_t yb = size_t(layer->shape.M) * (y_is_fp32 ? 4 : 2);
  if (ranges_overlap(d_x, xb, d_y, yb)) return fail(FLUXBIN_ERR_INVALID_ARG, "x and y overlap");
  return gemv_noalloc(*layer, d_x, d_y, y_is_fp32, stream);
}

fluxbin_status fluxbin_debug_indices(const fluxbin_layer* layer, uint8_t* d_p, hipStream_t stream) {
  g_msg[0] = 0;
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  if (!d_p) return fail(FLUXBIN_ERR_INVALID_ARG, "d_p is NULL");
  return launch_debug_indices(*layer, d_p, stream);
}

fluxbin_status fluxbin_unpack_canonical(const fluxbin_layer* layer, uint32_t* d_signs_out, uint32_t* d_dense_out,
                                        hipStream_t stream) {
  g_msg[0] = 0;
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  if (!d_signs_out) return fail(FLUXBIN_ERR_INVALID_ARG, "d_signs_out is NULL");
  return launch_unpack(*layer, d_signs_out, d_dense_out, stream);
}

fluxbin_status fluxbin_stream_probe(const fluxbin_layer* layer, uint32_t* d_sink, size_t sink_bytes,
                                    hipStream_t stream) {
  g_msg[0] = 0;
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  if (!d_sink) return fail(FLUXBIN_ERR_INVALID_ARG, "d_sink is NULL");
  if (sink_bytes < 1024) return fail(FLUXBIN_ERR_BUFFER_TOO_SMALL, "sink of %zu bytes < 1024", sink_bytes);
  Plan p;
  st = make_plan(*layer, 1, &p, false);
  if (st != FLUXBIN_OK) return st;
  if (p.kernel != 0)
    return fail(FLUXBIN_ERR_UNSUPPORTED, "the stream probe follows the split-tile batch-1 kernel's launch plan, and "
                                         "this layer runs kernel %d at batch 1", p.kernel);
  return launch_stream_probe(*layer, p, d_sink, stream);
}

fluxbin_status fluxbin_get_tuning(fluxbin_tuning* out) {
  g_msg[0] = 0;
  if (!out) return fail(FLUXBIN_ERR_INVALID_ARG, "out is NULL");
  *out = tuning_snapshot();
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_set_tuning(const fluxbin_tuning* t) {
  g_msg[0] = 0;
  std::lock_guard<std::mutex> lock(g_tuning_mu);
  g_tuning = t ? *t : tuning_defaults();
  g_tuning_init = true;
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_plan_query(const fluxbin_layer* layer, int32_t B, fluxbin_plan_info* out) {
  g_msg[0] = 0;
  fluxbin_status st = check_layer(layer);
  if (st != FLUXBIN_OK) return st;
  if (!out) return fail(FLUXBIN_ERR_INVALID_ARG, "out is NULL");
  if (B < 1 || B > kMaxBatchCall) return fail(FLUXBIN_ERR_INVALID_ARG, "B = %d out of range [1, %d]", B, kMaxBatchCall);
  BatchTiles bt;
  st = batch_tiles(*layer, B, batch_tile_rows(*layer, tuning_snapshot(), B), &bt);
  if (st != FLUXBIN_OK) return st;
  const Plan& p = bt.n_full > 0 ? bt.full : bt.tail;
  std::memset(out, 0, sizeof(*out));
  out->kernel = p.kernel;
  out->threads = p.nt;
  out->rows_per_tile = p.rows;
  out->depth = p.depth;
  out->batch_groups = p.n_groups;
  out->second_kernel_reduction = p.reduce2 ? 1 : 0;
  out->early = p.early ? 1 : 0;
  out->batch_tiles = bt.n_full + (bt.tail_rows > 0 ? 1 : 0);
  out->batch_tile_rows = bt.tile;
  out->workgroups_per_tile = p.kpt;
  out->tiles = p.n_tiles;
  out->units = p.units;
  out->workgroups = p.blocks;
  out->workspace_bytes = bt.ws_bytes;
  return FLUXBIN_OK;
}

}  // extern "C"

