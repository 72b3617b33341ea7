// Descriptors and launchers of the Shampoo owner step (fp32 throughout).
//
// Every matrix the step works on lives in the workspace as a zero-padded row-major fp32 buffer
// whose row and column counts are multiples of kShTile (128), so the GEMM needs no edge
// handling. Caller buffers (gradient, parameter, statistics, preconditioners) keep their natural
// m x n / m x m / n x n row-major layout; small copy kernels move data across that boundary.
//
// Zero padding is exact for every product: a padded statistic S is block diagonal (the real block
// and a zero block), the root iteration keeps that structure (products of block-diagonal matrices),
// and the padded rows and columns of the gradient are zero, so they add nothing to P_L G P_R.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfsdp {

constexpr int kShTile = 128;     // GEMM output tile and padding granularity
constexpr int kShCopyTile = 64;  // copy / init / apply tile
// Convergence of the inverse-root iteration: once max |M_k - I| over the real block is below this,
// the remaining change of X is below 2.5e-6 relative (T_k = I - (M_k - I)/p, then quadratic), and
// the side's remaining products are skipped.
constexpr float kShConvTol = 1e-5f;

// C = alpha * P Q^T + beta * E + diag * I over one padded problem (P: M x K, Q: N x K, all
// row-major with the given row strides; M, N and K multiples of kShTile). sym: only tiles bi <= bj are computed; each is stored at
// (bi, bj) and transposed at (bj, bi). E may alias C (each element is read before it is written,
// by the same thread).
struct ShGemmDesc {
  const float* P;
  const float* Q;
  const float* E;
  float* C;
  int64_t ldp, ldq, lde, ldc;
  int32_t K;
  int32_t tiles_n;     // N / kShTile (= M / kShTile when sym)
  int32_t sym;
  int32_t tile_begin;  // prefix over the problems of one launch
  float alpha, beta, diag;
  // inverse-root iteration only (null otherwise). Each side has two residual slots; iteration k
  // (parity q) reads slot q^1 (written by iteration k-1) and writes slot q:
  const float* conv_in;  // skip the product when this residual is below kShConvTol (and, with
                         // copy_on_skip, copy the tile of E into C instead)
  float* clear;          // set to 0 by the problem's first block before anything else
  float* resid_out;      // max |C - I| over the real block (rows, cols < valid), atomic max
  int32_t copy_on_skip;
  int32_t valid;
  // operand stored as bf16 (a bf16 gradient; row stride in elements): it is one part of the bf16
  // split, so the products with the zero mid and lo parts of an fp32 split are dropped. Both P and
  // Q, or Q alone (P alone is not supported). fp32 operands are split into three parts.
  int32_t p_bf16, q_bf16;
};

// Boundary copies over 64 x 64 tiles of a padded rows_pad x cols_pad domain.
// in  (dir 0): dst[r][c] = src[r][c] inside rows x cols, 0 elsewhere; optional dstT[c][r] too
//              (dst may be null when dstT is set); both fp32, or both bf16 when dst_bf16 (for a
//              bf16 source: the copy is exact).
// out (dir 1): dst (caller, rows x cols fp32, row stride ld_dst) = src (padded fp32) inside.
struct ShCopyDesc {
  const void* src;
  void* dst;
  void* dstT;
  int64_t rows, cols;
  int64_t ld_src, ld_dst, ld_dstT;
  int32_t src_dtype;   // kDtF32 / kDtBF16 (dir 0)
  int32_t tiles_n;     // column tiles of the domain
  int32_t tile_begin;
  int32_t dst_bf16;    // dir 0: dst and dstT hold bf16
};

// Sum of squares and trace of a padded d_pad x d_pad statistic, in row chunks (fp64 partials).
struct ShNormDesc {
  const float* S;
  int64_t ld;
  int32_t rows_pad;
  int32_t chunk_rows;
  double* partials;    // 2 doubles per chunk: (sum S^2, trace part)
  int32_t nchunks;
  int32_t tile_begin;  // first block of this problem in the launch
};

// Root scalars of one problem from its partials: rho = eps + eps_rel ||S||_F,
// z = (1 + p) / (2 ||S + rho I||_F) over the real dimension d; out = {rho, z, z^(1/p)}.
struct ShScalarDesc {
  const double* partials;
  int32_t nchunks;
  int32_t d;
  float* out;
};

// M = z (S + rho I), X = z^(1/p) I over the padded domain (the padded diagonal is rho as well).
struct ShInitDesc {
  const float* S;
  float* M;
  float* X;
  float* resid;        // the two residual slots: {0, not converged}
  int64_t ld;
  const float* sc;     // {rho, z, z^(1/p)}
  int32_t tiles_n;
  int32_t tile_begin;
};

// p <- p (1 - lr wd) - lr U (U padded fp32), and optionally update_out = U.
struct ShApplyDesc {
  const float* U;
  int64_t ldu;
  void* param;
  float* update_out;
  int64_t m, n;
  int32_t param_dtype;
  int32_t tiles_n;
  int32_t tile_begin;
};

hipError_t launch_sh_gemm(const ShGemmDesc* d, int count, int total_tiles, hipStream_t st);
hipError_t launch_sh_copy(const ShCopyDesc* d, int count, int total_tiles, int dir, hipStream_t st);
hipError_t launch_sh_norm(const ShNormDesc* d, int count, int total_blocks, hipStream_t st);
hipError_t launch_sh_scalars(const ShScalarDesc* d, int count, double eps, double eps_rel, int p,
                             hipStream_t st);
hipError_t launch_sh_init(const ShInitDesc* d, int count, int total_tiles, hipStream_t st);
hipError_t launch_sh_apply(const ShApplyDesc* d, int count, int total_tiles, float decay, float step,
                           hipStream_t st);

}  // namespace mfsdp
