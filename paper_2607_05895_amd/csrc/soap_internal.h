// Descriptors and launchers of the SOAP owner step and of its basis refresh (fp32 throughout).
//
// The products of the step run on the Shampoo GEMM (sh_gemm_kernel) over zero-padded row-major
// buffers (multiples of kShTile). The kernels declared here are the ones specific to SOAP: the
// first-moment pass, the Adam pass in the eigenbasis, and the pieces of the blocked Householder QR
// that refreshes a basis (16-column panel factorization, the panel's reflector applied to the rest
// of its 128-column block, and the block's compact-WY factor; the block's update of the trailing
// matrix and of the accumulated Q runs on the Shampoo GEMM).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "shampoo_internal.h"

namespace mfsdp {

constexpr int kQrPanel = 16;          // columns per Householder panel
constexpr int kQrBlock = 128;         // columns per block reflector (8 panels; the GEMM's tile)
constexpr int kQrPanelThreads = 512;  // one workgroup per panel (2 waves per SIMD: 256 registers each)
constexpr int kQrRowsPerThread = 8;   // panel rows held in registers per thread
constexpr int kQrMaxDim = kQrPanelThreads * kQrRowsPerThread;  // 4096
constexpr int kQrColThreads = 256;    // in-block application: one workgroup per column
constexpr int kQrColRows = kQrMaxDim / kQrColThreads;          // column entries per thread
constexpr int kQrGramChunk = 256;     // K chunk of the split V^T V product
static_assert(kQrBlock == kShTile, "the block update runs on the Shampoo GEMM's tiles");

// M <- beta1 M + (1 - beta1) G over the real m x n block, and the padded layouts the products read
// (each written only if its pointer is set): Gp (mp x np, row stride np) = G; GMt rows [0, np) = G^T
// and rows [np, 2 np) = M^T (row stride mp); GM (mp x 2 np, row stride 2 np) = [G | M] (a left side
// without a basis: the right product reads G and M as they are). With g_bf16 (a bf16 gradient) Gp
// and GMt's G^T rows hold bf16 (same row strides in elements; exact), for the GEMM's one-part
// operands; M^T stays fp32 at GMt + np mp, unless Mr is set: then M itself (row stride np) goes
// there instead (the right product first, for a wide matrix). 64 x 64 tiles over the padded
// mp x np domain; zeros outside the real block.
struct SoapPrepDesc {
  const void* grad;
  float* exp_avg;
  float* Gp;
  float* GMt;
  float* GM;
  float* Mr;
  int64_t m, n, mp, np;
  int32_t grad_dtype;
  int32_t tiles_n;
  int32_t tile_begin;
  int32_t g_bf16;
};

// Adam in the eigenbasis over the real block: GMr = [G' | M'] (mp x 2 np, row stride 2 np);
// V <- beta2 V + (1 - beta2) G'^2 (caller m x n), N' = (M' inv_bc1) / (sqrt(V) inv_sqrt_bc2 + eps),
// stored transposed into NpT (np x mp, row stride mp) for the left back-product, or as it is into Np
// (mp x np, row stride np) when the left side has no basis (each written only if its pointer is
// set; Np must not overlap GMr); zeros outside the real block.
struct SoapAdamDesc {
  const float* GMr;
  float* exp_avg_sq;
  float* NpT;
  float* Np;
  int64_t m, n, mp, np;
  int32_t tiles_n;
  int32_t tile_begin;
};

// X = I over the real d x d block of a padded dp x dp buffer (row stride ld), zero elsewhere.
struct SoapEyeDesc {
  float* X;
  int64_t ld;
  int64_t d, dp;
  int32_t tiles_n;
  int32_t tile_begin;
};

// The refresh factors A (d x d, real block of a padded dp x dp matrix) stored transposed: At is
// row-major with row stride ld and holds A^T, so column j of A is row j of At (contiguous). Each
// 128-column block [j0, j0 + 128) of A has its reflectors in V ((dp - j0) x 128, row-major, row 0 =
// A's row j0), the same transposed in Vt (128 x (dp - j0), row stride ldvt), and its compact-WY
// factor T (128 x 128 upper triangular, row-major), so that the block's reflectors multiply to
// H_1 ... H_128 = I - V T V^T (reflectors past the real dimension are the identity: zero columns of
// V, zero rows and columns of T).

// Householder factorization of panel s of a block: A's columns [c, c + jb) (c = j0 + 16 s), rows
// [c, d) (d - c <= kQrMaxDim; jb = min(16, d - c), 0 when c >= d). Writes the panel's 16 columns of V
// and rows of Vt over all dp - j0 block rows (zero above the pivot rows, 1 on them, zero below d and
// for columns >= jb) and its 16 x 16 factor into T's diagonal block s. A is only read (R is not
// needed).
struct QrPanelDesc {
  const float* At;
  int64_t ld;
  float* V;
  float* Vt;
  float* T;
  int64_t ldvt;
  int32_t j0, c, jb, d, vrows;  // vrows = dp - j0
};

// The reflectors of panel s applied to the block's later columns: x <- (I - V_s T_s^T V_s^T) x for
// every column x of A in [c + 16, c + 16 + ncols), over rows [c, d), with V_s the panel's 16
// columns of V and T_s its diagonal block of T. One workgroup per column.
struct QrColDesc {
  float* At;
  int64_t ld;
  const float* V;  // the panel's first column of V, at row c - j0 (row stride kQrBlock)
  const float* T;  // the panel's diagonal block of T (row stride kQrBlock)
  int32_t c, rows, ncols;
  int32_t tile_begin;  // first workgroup of this problem in the launch
};

// The block's factor T from its panels' diagonal blocks (already in T) and G = V^T V, given as nG
// partial sums (consecutive 128 x 128 row-major): for s = 1 .. 7,
// T[0:16s, 16s:16s+16] = -T[0:16s, 0:16s] G[0:16s, 16s:16s+16] T_s; zero below the diagonal blocks.
// One workgroup per block.
struct QrTDesc {
  float* T;
  const float* G;
  int32_t nG;
};

hipError_t launch_soap_prep(const SoapPrepDesc* d, int count, int total_tiles, float beta1,
                            hipStream_t st);
hipError_t launch_soap_adam(const SoapAdamDesc* d, int count, int total_tiles, float beta2, float eps,
                            float inv_bc1, float inv_sqrt_bc2, hipStream_t st);
hipError_t launch_soap_eye(const SoapEyeDesc* d, int count, int total_tiles, hipStream_t st);
hipError_t launch_qr_panel(const QrPanelDesc* d, int count, hipStream_t st);
hipError_t launch_qr_col(const QrColDesc* d, int count, int total_blocks, hipStream_t st);
hipError_t launch_qr_t(const QrTDesc* d, int count, hipStream_t st);

}  // namespace mfsdp
