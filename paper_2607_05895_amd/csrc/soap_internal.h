// Descriptors and launchers of the SOAP owner step and of its basis refresh (fp32 throughout).
//
// The products of the step run on the Shampoo GEMM (sh_gemm_kernel) over zero-padded row-major
// buffers (multiples of kShTile). The kernels declared here are the ones specific to SOAP: the
// first-moment pass, the Adam pass in the eigenbasis, and the blocked Householder QR that refreshes
// a basis (panel factorization + block-reflector application).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "shampoo_internal.h"

namespace mfsdp {

constexpr int kQrPanel = 16;          // columns per Householder panel
constexpr int kQrPanelThreads = 512;  // one workgroup per panel (2 waves per SIMD: 256 registers each)
constexpr int kQrRowsPerThread = 8;   // panel rows held in registers per thread
constexpr int kQrMaxDim = kQrPanelThreads * kQrRowsPerThread;  // 4096
constexpr int kQrApplyCols = 64;      // columns per block of the reflector application

// M <- beta1 M + (1 - beta1) G over the real m x n block, and the padded layouts the products read
// (each written only if its pointer is set): Gp (mp x np, row stride np) = G; GMt rows [0, np) = G^T
// and rows [np, 2 np) = M^T (row stride mp); GM (mp x 2 np, row stride 2 np) = [G | M] (a left side
// without a basis: the right product reads G and M as they are). 64 x 64 tiles over the padded
// mp x np domain; zeros outside the real block.
struct SoapPrepDesc {
  const void* grad;
  float* exp_avg;
  float* Gp;
  float* GMt;
  float* GM;
  int64_t m, n, mp, np;
  int32_t grad_dtype;
  int32_t tiles_n;
  int32_t tile_begin;
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

// X = I over the real d x d block of a padded buffer (row stride ld).
struct SoapEyeDesc {
  float* X;
  int64_t ld;
  int64_t d;
  int32_t tiles_n;
  int32_t tile_begin;
};

// Householder factorization of one panel: columns [j0, j0 + jb) of A, rows [j0, j0 + rows)
// (rows = d - j0 <= kQrMaxDim). Writes V (rows x 16, row-major: column k is v_k, zero above its
// pivot, 1 on it, zero for k >= jb) and T (16 x 16 upper triangular, H_1 ... H_jb = I - V T V^T).
// A is only read (R is not needed). The panel's 16 columns must lie inside A's row stride.
struct QrPanelDesc {
  const float* A;
  int64_t lda;
  float* V;
  float* T;
  int32_t j0, jb, rows;
};

// X <- (I - V T^T V^T) X on rows [row0, row0 + rows) and columns [c0, c0 + cols) of X: the panel's
// block reflector applied from the left, both to the trailing columns of the matrix being
// factored and to the accumulated Q^T.
struct QrApplyDesc {
  float* X;
  int64_t ldx;
  const float* V;
  const float* T;
  int32_t row0, rows;
  int32_t c0, cols;
  int32_t tile_begin;  // blocks of kQrApplyCols columns, prefix over the launch
};

hipError_t launch_soap_prep(const SoapPrepDesc* d, int count, int total_tiles, float beta1,
                            hipStream_t st);
hipError_t launch_soap_adam(const SoapAdamDesc* d, int count, int total_tiles, float beta2, float eps,
                            float inv_bc1, float inv_sqrt_bc2, hipStream_t st);
hipError_t launch_soap_eye(const SoapEyeDesc* d, int count, int total_tiles, hipStream_t st);
hipError_t launch_qr_panel(const QrPanelDesc* d, int count, hipStream_t st);
hipError_t launch_qr_apply(const QrApplyDesc* d, int count, int total_blocks, hipStream_t st);
// dst (caller, cols x rows, row stride ld_dst) = transpose of src (padded, rows x cols inside).
hipError_t launch_copy_out_transposed(const ShCopyDesc* d, int count, int total_tiles, hipStream_t st);

}  // namespace mfsdp
