// FluxBin weight decomposition on the GPU (fp64): RC_Decomp and StructuralSearch.
//
// RC_Decomp (App. algorithm "FluxBin Sub-routines"; Def. RC decomposition, Props. 3.2 and 3.3) approximates X * mask,
// block by block of g columns, by K binary bases W^(k) = (alpha_r^(k) alpha_c^(k)^T) * B^(k) with one row scale per
// (row, block) and one column scale per column:
//   greedy initialization: for k = 1..K: B^(k) = sign of the residual on the mask (sign(0) = +1), alpha_c^(k) = 1, one
//   row-scale and one column-scale least-squares update (Prop. 3.2), the residual loses the base's contribution;
//   T rounds of: for each base the row then the column scales by least squares against the target X * mask minus the
//   other bases' contributions; then every element's signs by exhaustive search over the 2^K combinations (Prop. 3.3),
//   first minimum in the order c = 0..2^K-1 (bit k of c set: b_k = +1); signs are 0 off the mask.
// StructuralSearch (Def. Hessian-based Column Saliency, with a diagonal inverse Hessian): S_j = sum_i W_ij^2 / h_j^2,
// and per block of g columns the s columns of largest saliency (equal scores: smaller column index first).
//
// Every step is a data-parallel kernel over the whole matrix (all blocks at once), launched in sequence on the stream.
// Sums use fixed reduction trees (no atomics), so results are deterministic. Arithmetic is fp64, the precision in which
// the integer sign decisions are taken.
#include <hip/hip_runtime.h>

#include "fluxbin_internal.h"

namespace fluxbin {

namespace {

struct RcArgs {
  const float* X;         // [M][N]
  const uint8_t* mask;    // [N] or nullptr (all columns)
  const uint32_t* pB;     // prior bases subtracted from X (canonical bit planes [Kp][M][ceil(N/32)]), or nullptr
  const double* par;      // [Kp][M][pG]
  const double* pac;      // [Kp][N]
  int32_t Kp;
  int64_t pg, pG, pW;
  int8_t* B;              // [K][M][N]
  double* ar;             // [K][M][G]
  double* ac;             // [K][N]
  int64_t M, N, g, G;
  int32_t K;
  double eps;
};

__device__ __forceinline__ bool rc_in(const RcArgs& a, int64_t j) { return a.mask == nullptr || a.mask[j] != 0; }

// The matrix being decomposed at (i, j), before the mask: X, or X minus the prior bases' approximation (the residual of
// an earlier decomposition, FluxBin-Hybrid step 3), the prior contributions summed first in base order.
__device__ __forceinline__ double rc_x(const RcArgs& a, int64_t i, int64_t j) {
  const double x = double(a.X[i * a.N + j]);
  if (a.pB == nullptr) return x;
  double s = 0.0;
  for (int p = 0; p < a.Kp; ++p) {
    const double m = a.par[(p * a.M + i) * a.pG + j / a.pg] * a.pac[p * a.N + j];
    const bool plus = (a.pB[(p * a.M + i) * a.pW + (j >> 5)] >> (j & 31)) & 1u;
    s += plus ? m : -m;
  }
  return x - s;
}

__device__ __forceinline__ double rc_contrib(const RcArgs& a, int kk, int64_t i, int64_t j) {
  const double m = a.ar[(kk * a.M + i) * a.G + j / a.g] * a.ac[kk * a.N + j];
  return m * double(a.B[(kk * a.M + i) * a.N + j]);
}

// Target of base k at (i, j). Initialization (init != 0): the residual after bases 0..k-1, subtracted one by one.
// Rounds: X * mask minus the sum of the other bases' contributions (summed first, in base order).
__device__ __forceinline__ double rc_target(const RcArgs& a, int k, int init, int64_t i, int64_t j) {
  const double x = rc_in(a, j) ? rc_x(a, i, j) : 0.0;
  if (init) {
    double r = x;
    for (int kk = 0; kk < k; ++kk) r -= rc_contrib(a, kk, i, j);
    return r;
  }
  double s = 0.0;
  for (int kk = 0; kk < a.K; ++kk)
    if (kk != k) s += rc_contrib(a, kk, i, j);
  return x - s;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__global__ void k_rc_fill(double* p, int64_t n, double v) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// Greedy initialization of base k's signs: sign of the residual after bases 0..k-1 on the mask, 0 off it.
__global__ void k_rc_init_sign(RcArgs a, int k) {
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= a.M * a.N) return;
  const int64_t i = e / a.N, j = e - i * a.N;
  int8_t b = 0;
  if (rc_in(a, j)) b = rc_target(a, k, 1, i, j) >= 0.0 ? int8_t(1) : int8_t(-1);
  a.B[(int64_t(k) * a.M + i) * a.N + j] = b;
}

// Row scales of base k (Prop. 3.2): one wavefront per (row, block), lanes over the block's columns.
__global__ void __launch_bounds__(256) k_rc_row(RcArgs a, int k, int init) {
  const int64_t wid = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wid >= a.M * a.G) return;   // whole wavefronts leave together
  const int64_t i = wid / a.G, blk = wid - i * a.G;
  const int64_t c0 = blk * a.g, c1 = c0 + a.g < a.N ? c0 + a.g : a.N;
  double num = 0.0, den = 0.0;
  for (int64_t j = c0 + lane; j < c1; j += 64) {
    const double cb = a.ac[int64_t(k) * a.N + j] * double(a.B[(int64_t(k) * a.M + i) * a.N + j]);
    num += cb * rc_target(a, k, init, i, j);
    den += cb * cb;
  }
  num = wave_sum(num);
  den = wave_sum(den);
  if (lane == 0) a.ar[(int64_t(k) * a.M + i) * a.G + blk] = num / (den + a.eps);
}

// Column scales of base k (Prop. 3.2), first stage: workgroup (tile of 64 columns, row slice r of RS) sums its rows
// in four interleaved sub-slices combined in a fixed order, into part[r][2][N] (numerator, denominator).
__global__ void __launch_bounds__(256) k_rc_col(RcArgs a, int k, int init, int64_t rows_per_slice, double* part) {
  __shared__ double s_num[4][64], s_den[4][64];
  const int c = threadIdx.x & 63, sub = threadIdx.x >> 6;
  const int64_t j = int64_t(blockIdx.x) * 64 + c;
  const int64_t r = blockIdx.y;
  const int64_t i0 = r * rows_per_slice, i1 = i0 + rows_per_slice < a.M ? i0 + rows_per_slice : a.M;
  double num = 0.0, den = 0.0;
  if (j < a.N) {
    const int64_t blk = j / a.g;
    for (int64_t i = i0 + sub; i < i1; i += 4) {
      const double rb = a.ar[(int64_t(k) * a.M + i) * a.G + blk] * double(a.B[(int64_t(k) * a.M + i) * a.N + j]);
      num += rb * rc_target(a, k, init, i, j);
      den += rb * rb;
    }
  }
  s_num[sub][c] = num;
  s_den[sub][c] = den;
  __syncthreads();
  if (sub == 0 && j < a.N) {
    part[(r * 2 + 0) * a.N + j] = ((s_num[0][c] + s_num[1][c]) + s_num[2][c]) + s_num[3][c];
    part[(r * 2 + 1) * a.N + j] = ((s_den[0][c] + s_den[1][c]) + s_den[2][c]) + s_den[3][c];
  }
}

// Second stage: the slices' sums added in slice order, then the least-squares quotient.
__global__ void k_rc_col_fin(RcArgs a, int k, int64_t slices, const double* part) {
  const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= a.N) return;
  double n = 0.0, d = 0.0;
  for (int64_t r = 0; r < slices; ++r) {
    n += part[(r * 2 + 0) * a.N + j];
    d += part[(r * 2 + 1) * a.N + j];
  }
  a.ac[int64_t(k) * a.N + j] = n / (d + a.eps);
}

// Joint sign search (Prop. 3.3) for every element: the first of the 2^K combinations with the smallest |x - approx|.
template <int K>
__global__ void k_rc_sign(RcArgs a) {
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= a.M * a.N) return;
  const int64_t i = e / a.N, j = e - i * a.N;
  const bool in = rc_in(a, j);
  const double x = in ? rc_x(a, i, j) : 0.0;
  const int64_t blk = j / a.g;
  double m[K];
#pragma unroll
  for (int k = 0; k < K; ++k) m[k] = a.ar[(int64_t(k) * a.M + i) * a.G + blk] * a.ac[int64_t(k) * a.N + j];
  double best = 0.0;
  int best_c = -1;
#pragma unroll
  for (int c = 0; c < (1 << K); ++c) {
    double approx = 0.0;
#pragma unroll
    for (int k = 0; k < K; ++k) approx += ((c >> k) & 1) ? m[k] : -m[k];
    const double err = fabs(x - approx);
    if (best_c < 0 || err < best) {
      best = err;
      best_c = c;
    }
  }
#pragma unroll
  for (int k = 0; k < K; ++k)
    a.B[(int64_t(k) * a.M + i) * a.N + j] = in ? (((best_c >> k) & 1) ? int8_t(1) : int8_t(-1)) : int8_t(0);
}

// Signs to canonical planes [K][M][ceil(N/32)]: bit t of word w is B[k][i][32w + t] == +1.
__global__ void k_rc_bits(RcArgs a, uint32_t* out) {
  const int64_t W = (a.N + 31) / 32;
  const int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= int64_t(a.K) * a.M * W) return;
  const int64_t row = e / W, w = e - row * W;   // row = k * M + i
  uint32_t bits = 0u;
  for (int t = 0; t < 32; ++t) {
    const int64_t j = w * 32 + t;
    if (j < a.N && a.B[row * a.N + j] == 1) bits |= 1u << t;
  }
  out[e] = bits;
}

// Column saliency S_j = sum_i W_ij^2 / h_j^2: a workgroup per 64 columns, four row slices combined in a fixed order.
__global__ void __launch_bounds__(256) k_saliency(const float* W, const double* h, int64_t M, int64_t N, double* S) {
  __shared__ double s_sum[4][64];
  const int c = threadIdx.x & 63, slice = threadIdx.x >> 6;
  const int64_t j = int64_t(blockIdx.x) * 64 + c;
  double acc = 0.0;
  if (j < N)
    for (int64_t i = slice; i < M; i += 4) {
      const double w = double(W[i * N + j]);
      acc += w * w;
    }
  s_sum[slice][c] = acc;
  __syncthreads();
  if (slice == 0 && j < N) S[j] = (((s_sum[0][c] + s_sum[1][c]) + s_sum[2][c]) + s_sum[3][c]) / (h[j] * h[j]);
}

// Per block of g columns (a workgroup each, g <= 1024): column j is selected when fewer than s columns of the block
// rank before it (larger score, or equal score and smaller index); the selected columns are written in increasing
// index order after the min(s, g) columns of every earlier block.
__global__ void __launch_bounds__(1024) k_topk(const double* S, int64_t N, int64_t g, int64_t s, int32_t* idx,
                                               uint8_t* mask) {
  __shared__ double sc[1024];
  __shared__ int sel[1024];
  const int64_t c0 = int64_t(blockIdx.x) * g;
  const int n = int(c0 + g < N ? g : N - c0);
  const int t = threadIdx.x;
  if (t < n) sc[t] = S[c0 + t];
  __syncthreads();
  int chosen = 0;
  if (t < n) {
    int rank = 0;
    for (int u = 0; u < n; ++u) rank += (sc[u] > sc[t] || (sc[u] == sc[t] && u < t)) ? 1 : 0;
    chosen = rank < s ? 1 : 0;
  }
  sel[t] = chosen;
  if (mask != nullptr && t < n) mask[c0 + t] = uint8_t(chosen);
  __syncthreads();
  if (t < n && chosen) {
    int before = 0;
    for (int u = 0; u < t; ++u) before += sel[u];
    idx[int64_t(blockIdx.x) * s + before] = int32_t(c0 + t);
  }
}

unsigned grid_for(int64_t n, int per) { return unsigned((n + per - 1) / per); }

// Row slices of the column-scale sums: at least 256 rows each, at most 64 slices.
int64_t col_slices(int64_t M) {
  const int64_t s = M / 256;
  return s < 1 ? 1 : (s > 64 ? 64 : s);
}

}  // namespace

}  // namespace fluxbin

using namespace fluxbin;

extern "C" {

fluxbin_status fluxbin_rc_workspace_query(int64_t M, int64_t N, int32_t K, size_t* bytes) {
  clear_error();
  if (!bytes) return fail(FLUXBIN_ERR_INVALID_ARG, "bytes is NULL");
  if (M < 1 || N < 1 || K < 1 || K > 4) return fail(FLUXBIN_ERR_INVALID_ARG, "M, N >= 1 and K in 1..4 required");
  // int8 signs [K][M][N], then (256-byte aligned) the column-scale partial sums [slices][2][N] fp64
  *bytes = ((size_t(K) * size_t(M) * size_t(N) + 255) & ~size_t(255)) + size_t(col_slices(M)) * 2 * size_t(N) * 8;
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_rc_decompose(const float* d_X, const uint8_t* d_mask, const uint32_t* d_prior_signs,
                                    const double* d_prior_alpha_r, const double* d_prior_alpha_c, int32_t Kp,
                                    int64_t gp, int64_t M, int64_t N, int32_t K, int32_t T, int64_t g, double eps,
                                    uint32_t* d_signs, double* d_alpha_r, double* d_alpha_c, void* d_ws,
                                    size_t ws_bytes, hipStream_t stream) {
  size_t need = 0;
  fluxbin_status st = fluxbin_rc_workspace_query(M, N, K, &need);
  if (st != FLUXBIN_OK) return st;
  if (!d_X || !d_signs || !d_alpha_r || !d_alpha_c || !d_ws)
    return fail(FLUXBIN_ERR_INVALID_ARG, "a required pointer is NULL");
  if (T < 0 || g < 1 || !(eps >= 0.0)) return fail(FLUXBIN_ERR_INVALID_ARG, "T >= 0, g >= 1 and eps >= 0 required");
  if (d_prior_signs && (!d_prior_alpha_r || !d_prior_alpha_c || Kp < 1 || Kp > 4 || gp < 1))
    return fail(FLUXBIN_ERR_INVALID_ARG, "prior bases need their scales, Kp in 1..4 and gp >= 1");
  if (M * N > (int64_t(1) << 36)) return fail(FLUXBIN_ERR_UNSUPPORTED, "matrix of %lld elements too large",
                                              (long long)(M * N));
  if (ws_bytes < need)
    return fail(FLUXBIN_ERR_BUFFER_TOO_SMALL, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  RcArgs a{};
  a.X = d_X;
  a.mask = d_mask;
  a.B = static_cast<int8_t*>(d_ws);
  a.ar = d_alpha_r;
  a.ac = d_alpha_c;
  a.M = M;
  a.N = N;
  a.g = g;
  a.G = (N + g - 1) / g;
  a.K = K;
  a.eps = eps;
  a.pB = d_prior_signs;
  a.par = d_prior_alpha_r;
  a.pac = d_prior_alpha_c;
  a.Kp = d_prior_signs ? Kp : 0;
  a.pg = d_prior_signs ? gp : 1;
  a.pG = (N + a.pg - 1) / a.pg;
  a.pW = (N + 31) / 32;
  const int64_t elems = M * N;
  const int64_t slices = col_slices(M);
  const int64_t rows_per_slice = (M + slices - 1) / slices;
  double* part = reinterpret_cast<double*>(static_cast<char*>(d_ws) +
                                           ((size_t(K) * size_t(M) * size_t(N) + 255) & ~size_t(255)));
  const dim3 col_grid(grid_for(N, 64), unsigned(slices));
  for (int k = 0; k < K; ++k) {
    hipLaunchKernelGGL(k_rc_fill, dim3(grid_for(N, 256)), dim3(256), 0, stream, d_alpha_c + int64_t(k) * N, N, 1.0);
    hipLaunchKernelGGL(k_rc_init_sign, dim3(grid_for(elems, 256)), dim3(256), 0, stream, a, k);
    hipLaunchKernelGGL(k_rc_row, dim3(grid_for(M * a.G, 4)), dim3(256), 0, stream, a, k, 1);
    hipLaunchKernelGGL(k_rc_col, col_grid, dim3(256), 0, stream, a, k, 1, rows_per_slice, part);
    hipLaunchKernelGGL(k_rc_col_fin, dim3(grid_for(N, 256)), dim3(256), 0, stream, a, k, slices, part);
  }
  for (int t = 0; t < T; ++t) {
    for (int k = 0; k < K; ++k) {
      hipLaunchKernelGGL(k_rc_row, dim3(grid_for(M * a.G, 4)), dim3(256), 0, stream, a, k, 0);
      hipLaunchKernelGGL(k_rc_col, col_grid, dim3(256), 0, stream, a, k, 0, rows_per_slice, part);
      hipLaunchKernelGGL(k_rc_col_fin, dim3(grid_for(N, 256)), dim3(256), 0, stream, a, k, slices, part);
    }
    switch (K) {
      case 1: hipLaunchKernelGGL(k_rc_sign<1>, dim3(grid_for(elems, 256)), dim3(256), 0, stream, a); break;
      case 2: hipLaunchKernelGGL(k_rc_sign<2>, dim3(grid_for(elems, 256)), dim3(256), 0, stream, a); break;
      case 3: hipLaunchKernelGGL(k_rc_sign<3>, dim3(grid_for(elems, 256)), dim3(256), 0, stream, a); break;
      default: hipLaunchKernelGGL(k_rc_sign<4>, dim3(grid_for(elems, 256)), dim3(256), 0, stream, a); break;
    }
  }
  const int64_t words = int64_t(K) * M * ((N + 31) / 32);
  hipLaunchKernelGGL(k_rc_bits, dim3(grid_for(words, 256)), dim3(256), 0, stream, a, d_signs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the decomposition kernels");
  return FLUXBIN_OK;
}

fluxbin_status fluxbin_structural_search(const float* d_W, const double* d_hinv_diag, int64_t M, int64_t N,
                                         int64_t g, int64_t s, double* d_scores, int32_t* d_sal_idx,
                                         uint8_t* d_mask, hipStream_t stream) {
  clear_error();
  if (!d_W || !d_hinv_diag || !d_scores || !d_sal_idx) return fail(FLUXBIN_ERR_INVALID_ARG, "a pointer is NULL");
  if (M < 1 || N < 1 || g < 1 || s < 1) return fail(FLUXBIN_ERR_INVALID_ARG, "M, N, g, s >= 1 required");
  if (g > 1024) return fail(FLUXBIN_ERR_UNSUPPORTED, "group of %lld columns > 1024", (long long)g);
  if (s > g) return fail(FLUXBIN_ERR_INVALID_ARG, "s = %lld > g = %lld", (long long)s, (long long)g);
  if (M * N > (int64_t(1) << 36)) return fail(FLUXBIN_ERR_UNSUPPORTED, "matrix too large");
  hipLaunchKernelGGL(k_saliency, dim3(grid_for(N, 64)), dim3(256), 0, stream, d_W, d_hinv_diag, M, N, d_scores);
  hipLaunchKernelGGL(k_topk, dim3(unsigned((N + g - 1) / g)), dim3(1024), 0, stream, d_scores, N, g, s, d_sal_idx,
                     d_mask);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "launching the saliency kernels");
  return FLUXBIN_OK;
}

}  // extern "C"
