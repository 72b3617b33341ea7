// Internal descriptors and kernel launchers shared by the host library and the HIP kernels.
//
// Data layout in HBM for one Muon entry with stored shape m x n (r = min, s = max):
//   the NS iterate is kept in both layouts, zero padded to the NS tile size:
//     X[0], X[1]   r_pad x s_pad   (K = s_pad columns)   -- ping-pong over NS steps
//     XT[0], XT[1] s_pad x r_pad   (K = r_pad)           -- X^T of the same iterate
//     G            r_pad x r_pad   A = X X^T (symmetric)
//     H            r_pad x r_pad   B' = b A + c A A + a I (symmetric)
//   Zero padding is exact for the iteration: padded rows/columns of X give zero rows/columns of
//   A and B', and stay zero in B' X.
//   Every NS product is then an "NT" product C = P Q^T with both operands K-contiguous:
//     Gram      A = X X^T             P = Q = X,  K = s_pad
//     square    A A = A A^T           P = Q = A,  K = r_pad   (A symmetric)
//     update    B' X = B' (X^T)^T     P = B', Q = X^T, K = r_pad
//   The square product stores B' = c A A + b A + a I, so the update X' = a X + B X = B' X is a plain
//   product with no addend. It writes X' in both layouts so the next step again reads
//   K-contiguous operands.
//
//   All of these buffers are panel blocked (blk_index below): rows in blocks of 16, columns in
//   blocks of 32, each 16 x 32 block contiguous (1 KiB in bf16), the blocks of one 16-row panel
//   following each other along K. One K step of a 16-row slice of an operand is then one
//   contiguous KiB, which the GEMM's direct-to-LDS loads fetch as eight whole 128-B lines.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm_schedule.h"

namespace mfsdp {

// Element (r, k) of a panel-blocked buffer with K columns (K a multiple of 32, rows a multiple of
// 16). Eight consecutive k starting at a multiple of 8 are contiguous.
constexpr int kBlkRows = 16;
constexpr int kBlkCols = 32;
__host__ __device__ constexpr int64_t blk_index(int64_t r, int64_t k, int64_t K) {
  return (r >> 4) * (K << 4) + ((k >> 5) << 9) + ((r & 15) << 5) + (k & 31);
}

// Two floats to packed bf16 (lo in bits 0..15), round to nearest even, one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

constexpr int kDtF32 = 0;
constexpr int kDtBF16 = 1;

// ---------------------------------------------------------------------------------------------
// prep: momentum EMA + Nesterov (or a plain copy for standalone NS), Sum u^2 partials, and the
// NS input written in both layouts. One 64 x 64 tile of the stored m x n matrix per workgroup.
constexpr int kMaxGradParts = 64;

struct PrepDesc {
  const void* grad;      // m x n, grad_dtype (the NS input for standalone NS); unused if nparts > 0
  float* momentum;       // m x n fp32, or null for standalone NS
  void* d_out;           // u in stored orientation, padded, panel blocked with ld_d columns
  void* t_out;           // u^T, panel blocked with ld_t columns (ns dtype)
  float* partials;       // one Sum u^2 per tile
  int64_t m, n;          // stored shape
  int64_t ld_d, ld_t;
  int32_t tiles_m, tiles_n;  // over the padded domain, 64 x 64
  int32_t grad_dtype;
  int32_t tile_begin;    // first global tile index of this entry
  // owner-side reduction: g = gscale * (parts[0] + ... + parts[nparts - 1]) in fp32, in that order,
  // optionally stored to gout (grad_dtype); nparts == 0 reads grad instead
  int32_t nparts;
  float gscale;
  void* gout;
  const void* parts[kMaxGradParts];
};

// norm finalize: scale = 1 / max(sqrt(Sum partials), eps), deterministic order.
struct NormDesc {
  const float* partials;
  int32_t count;
  float* scale;
};

// apply: p <- p (1 - lr wd) - lr f (oscale O), or out <- oscale O for standalone NS.
struct ApplyDesc {
  const void* o;         // O in stored orientation (ns dtype), panel blocked with ld_o columns
  void* param;           // m x n, param dtype (or NS output)
  float* update_out;     // optional fp32 m x n
  const float* scale;    // norm scale, applied when no NS step ran (K = 0)
  int64_t m, n, ld_o;
  int32_t param_dtype;
  int32_t use_scale;
  int32_t mode;          // 0 = Muon parameter update, 1 = write O to param (standalone NS)
  float decay;           // 1 - lr wd
  float step;            // lr f
  int32_t tiles_m, tiles_n;
  int32_t tile_begin;
};

// Grouped NT GEMM problem: C = alpha * P Q^T + beta * E, stored in C and/or transposed in CT.
// Every operand is panel blocked; the ld* fields are the column counts. Both ping-pong alternatives are kept, indexed by step parity.
struct GemmDesc {
  const void* P[2];
  const void* Q[2];
  const void* E[2];
  void* C[2];
  void* CT[2];
  const float* scale;    // per-matrix norm scale (used on the first NS step), may be null
  int64_t ldp, ldq, lde, ldc, ldct;
  int32_t M, N, K;       // padded sizes, multiples of the tile
  float alpha, beta;     // (the square product takes its coefficients per launch instead)
  int32_t alpha_scale_pow;  // on the first step alpha *= scale^pow
  int32_t beta_scale_pow;
  int32_t sym;           // 1: only tiles bi <= bj, stored to (bi,bj) and mirrored to (bj,bi)
  int32_t tiles_m, tiles_n;
  int32_t tile_begin;    // prefix over the problems of one launch
  int32_t tile_count;
  int32_t last_c, last_ct;  // on the last step: write C / CT (1) or skip (0)
  // bf16 update product only: on the last step, apply the parameter update (or write the
  // standalone NS output) from the fp32 accumulators instead of storing the final iterate
  const ApplyDesc* fused;
  // bf16 Gram product with a split contraction (nks > 1): tile (bi, bj, range ks) stores its fp32
  // partial product in part (one 256 x 256 row-major tile per upper tile and range, at
  // ((upper index of (bi, bj)) * nks + ks) * 65536 floats) and a second pass adds the ranges in
  // order and stores A; 0 or 1: not split
  float* part;
  int32_t nks;
};
// Upper index of tile (bi, bj), bi <= bj, of a symmetric problem with tm tiles per side (row-major
// over the upper triangle).
__host__ __device__ constexpr int upper_index(int bi, int bj, int tm) { return bi * tm - bi * (bi - 1) / 2 + (bj - bi); }

constexpr int kAdamWMaxPerLaunch = 32;
struct AdamWDesc {
  void* param;
  const void* grad;
  float* exp_avg;
  float* exp_avg_sq;
  int64_t numel;
  int32_t param_dtype, grad_dtype;
  int32_t block_begin;
};
struct AdamWBatch {
  AdamWDesc d[kAdamWMaxPerLaunch];
  int32_t count;
  float decay;           // 1 - lr wd
  float beta1, beta2;
  float omb1, omb2;      // 1 - beta1, 1 - beta2 (formed in double)
  float step_size;       // lr / (1 - beta1^t)
  float inv_sqrt_bc2;    // 1 / sqrt(1 - beta2^t)
  float eps;
};
constexpr int kAdamWBlockElems = 2048;

// Launchers (return hipError_t of the launch).
// reduce: the descriptors' gradients are reductions of gradient parts (nparts >= 1 for all)
hipError_t launch_prep(const PrepDesc* d_descs, int count, int total_tiles, int ns_dtype,
                       int reduce, float beta, float one_minus_beta, int nesterov, hipStream_t st);
hipError_t launch_norm(const NormDesc* d_descs, int count, float eps, hipStream_t st);
// product: 0 Gram, 1 square, 2 update (the order of the products in one NS step); 3 the last update
// of the bf16 path with the fused parameter update (its descriptors carry `fused`)
// (ca, cb, cc): the NS step's coefficients (a_k, b_k, c_k), used by the square product.
// tile: the bf16 path's output tile, kTileBF16 or (Gram and square products only) kTileBF16Small;
// the descriptors' tile grids and the schedule are in that tile.
hipError_t launch_gemm(const GemmDesc* d_descs, int count, int total_tiles, const TileRef* d_sched,
                       int ngroups, int ns_dtype, int product, int parity, int first_step,
                       int last_step, float ca, float cb, float cc, int tile, hipStream_t st);
hipError_t launch_apply(const ApplyDesc* d_descs, int count, int total_tiles, int ns_dtype,
                        hipStream_t st);
// The second pass of a split Gram product: for each job (problem e in the Gram launch's order,
// upper tile bi <= bj) the problem's nks partial tiles added in range order, scaled as the Gram
// epilogue scales, stored as A (bf16) at (bi, bj) and mirrored at (bj, bi).
hipError_t launch_gram_sum(const GemmDesc* d_descs, const TileRef* d_jobs, int njobs, int parity,
                           int first, int tile, hipStream_t st);
hipError_t launch_adamw(const AdamWBatch& batch, int total_blocks, hipStream_t st);

// NS tile sizes (padding granularity of the workspace buffers).
constexpr int kTileBF16 = 256;
// The bf16 Gram and square products of a launch with few 256 x 256 tiles run on 128 x 128 tiles,
// two workgroups per CU (the padding stays 256).
constexpr int kTileBF16Small = 128;
constexpr int kTileF32 = 64;
constexpr int kPrepRows = 64;                    // prep tile rows
constexpr int kPrepColsBF16 = 256;              // prep tile columns on the bf16 path (divides 256)
constexpr int kPrepColsF32 = 64;                 // prep tile columns on the fp32 path
constexpr int kApplyCols = 128;                 // apply tile columns (8 per thread per row)
constexpr int kApplyRows = 16384 / kApplyCols;  // 16 K elements per tile: 64 per thread

}  // namespace mfsdp
