// HIP kernels specific to the SOAP owner step (fp32): the first-moment pass that also lays out the
// gradient for the products, Adam in the eigenbasis, and the blocked Householder QR that refreshes
// a basis. The products themselves run on the Shampoo GEMM.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "mfsdp_internal.h"
#include "soap_internal.h"

namespace mfsdp {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) float g_f32;
typedef __attribute__((address_space(1))) const float g_cf32;
typedef __attribute__((address_space(1))) f32x4 g_f32x4;
typedef __attribute__((address_space(1))) const f32x4 g_cf32x4;

constexpr int kTile = kShCopyTile;  // 64 x 64 tiles of the elementwise passes

template <typename D>
__device__ __forceinline__ int find_desc(const D* d, int count, int b) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (d[mid].tile_begin <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Compile-time loop: f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), so that
// register arrays indexed by the loop variable stay in registers.
template <typename F, int... I>
__device__ __forceinline__ void unrolled_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void unrolled(F&& f) {
  unrolled_impl(f, std::make_integer_sequence<int, N>{});
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes of a wave (all lanes active), the same value in every lane, in a fixed
// order: DPP butterflies within each 16-lane row (quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror, row_mirror: every lane of a row then holds the row sum; the partners' adds are
// commutative, so all lanes agree bit for bit), then the four row sums read from lanes 0, 16, 32,
// 48 and added in that order.
__device__ __forceinline__ float wave_sum(float x) {
  x += dpp<0xB1>(x);
  x += dpp<0x4E>(x);
  x += dpp<0x141>(x);
  x += dpp<0x140>(x);
  const int xi = __float_as_int(x);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(xi, 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(xi, 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(xi, 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(xi, 48));
  return ((r0 + r1) + r2) + r3;
}

// Sum of x over the four 16-lane rows of a wave, in every lane of the same column (all lanes
// active): rows 0 + 1 and 2 + 3 by swapping odd and even rows, then the two halves by swapping them
// (v_permlane16_swap, v_permlane32_swap: vector ALU exchanges, no LDS round trip). Each add has the
// same two operands in every lane that forms it, so all lanes of a column agree bit for bit.
__device__ __forceinline__ float sum_rows4(float x) {
  const uint32_t xi = __float_as_uint(x);
  const auto p = __builtin_amdgcn_permlane16_swap(xi, xi, false, false);
  const float y = __uint_as_float(p[0]) + __uint_as_float(p[1]);  // (row 2k) + (row 2k + 1)
  const uint32_t yi = __float_as_uint(y);
  const auto q = __builtin_amdgcn_permlane32_swap(yi, yi, false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);  // (rows 0, 1) + (rows 2, 3)
}

// Reduce-scatter of 16 values over the 16 lanes of a DPP row (all lanes active): afterwards lane l
// of each row holds that row's sum of value l (l = lane mod 16). Four exchange rounds with the lane
// at distance 1, 2, 4 and 8 (quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_shl/row_shr 4,
// row_ror 8): each lane keeps the half of its values whose index bit matches its own lane bit and
// adds the partner's copy of them; every sum is formed by exactly one lane, in a fixed order.
__device__ __forceinline__ float row_reduce_scatter16(const float (&v)[16], int l16) {
  const bool b0 = l16 & 1, b1 = (l16 >> 1) & 1, b2 = (l16 >> 2) & 1, b3 = (l16 >> 3) & 1;
  float s1[8], s2[4], s3[2];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float keep = b0 ? v[2 * j + 1] : v[2 * j], send = b0 ? v[2 * j] : v[2 * j + 1];
    s1[j] = keep + dpp<0xB1>(send);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float keep = b1 ? s1[2 * j + 1] : s1[2 * j], send = b1 ? s1[2 * j] : s1[2 * j + 1];
    s2[j] = keep + dpp<0x4E>(send);
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float keep = b2 ? s2[2 * j + 1] : s2[2 * j], send = b2 ? s2[2 * j] : s2[2 * j + 1];
    const float from_up = dpp<0x104>(send);    // row_shl 4: lane l reads lane l + 4
    const float from_down = dpp<0x114>(send);  // row_shr 4: lane l reads lane l - 4
    s3[j] = keep + (b2 ? from_down : from_up);
  }
  const float keep = b3 ? s3[1] : s3[0], send = b3 ? s3[0] : s3[1];
  return keep + dpp<0x128>(send);  // row_ror 8: lane l reads lane l ^ 8
}

__global__ __launch_bounds__(256) void soap_prep_kernel(const SoapPrepDesc* __restrict__ descs, int count,
                                                        float beta1) {
  __shared__ float tg[kTile][kTile + 1];
  __shared__ float tm[kTile][kTile + 1];
  const int e = find_desc(descs, count, blockIdx.x);
  const SoapPrepDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  const int64_t gc = int64_t(tj) * kTile + c;
  typedef __attribute__((address_space(1))) uint16_t g_u16;
  g_f32* Gp = (g_f32*)(d.Gp);
  g_f32* GMt = (g_f32*)(d.GMt);
  g_f32* GM = (g_f32*)(d.GM);
  g_f32* Mr = (g_f32*)(d.Mr);
  // G (and G^T) as bf16: the value's upper 16 bits, exact for a bf16 gradient
  auto put_g = [&](g_f32* base, int64_t i, float v) {
    if (d.g_bf16) ((g_u16*)base)[i] = uint16_t(__float_as_uint(v) >> 16);
    else base[i] = v;
  };
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;
    const int64_t gr = int64_t(ti) * kTile + r;
    float g = 0.0f, mo = 0.0f;
    if (gr < d.m && gc < d.n) {
      const int64_t o = gr * d.n + gc;
      g = d.grad_dtype == kDtBF16
              ? __uint_as_float(uint32_t(static_cast<const uint16_t*>(d.grad)[o]) << 16)
              : static_cast<const float*>(d.grad)[o];
      mo = beta1 * d.exp_avg[o] + (1.0f - beta1) * g;
      d.exp_avg[o] = mo;
    }
    if (Gp) put_g(Gp, gr * d.np + gc, g);
    if (Mr) Mr[gr * d.np + gc] = mo;
    if (GM) {
      GM[gr * 2 * d.np + gc] = g;
      GM[gr * 2 * d.np + d.np + gc] = mo;
    }
    tg[r][c] = g;
    tm[r][c] = mo;
  }
  if (!GMt) return;  // (uniform over the workgroup: no barrier is skipped by part of it)
  __syncthreads();
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;  // row of the transposed tile = column of the source tile
    const int64_t o = (int64_t(tj) * kTile + r) * d.mp + int64_t(ti) * kTile + c;
    put_g(GMt, o, tg[c][r]);
    if (!Mr) GMt[o + d.np * d.mp] = tm[c][r];
  }
}

__global__ __launch_bounds__(256) void soap_adam_kernel(const SoapAdamDesc* __restrict__ descs, int count,
                                                        float beta2, float eps, float inv_bc1,
                                                        float inv_sqrt_bc2) {
  __shared__ float tn[kTile][kTile + 1];
  const int e = find_desc(descs, count, blockIdx.x);
  const SoapAdamDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  const int64_t gc = int64_t(tj) * kTile + c;
  const g_cf32* GMr = (const g_cf32*)(d.GMr);
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;
    const int64_t gr = int64_t(ti) * kTile + r;
    float np_ = 0.0f;
    if (gr < d.m && gc < d.n) {
      const float gq = GMr[gr * 2 * d.np + gc];
      const float mq = GMr[gr * 2 * d.np + d.np + gc];
      const int64_t o = gr * d.n + gc;
      const float v = beta2 * d.exp_avg_sq[o] + (1.0f - beta2) * (gq * gq);
      d.exp_avg_sq[o] = v;
      np_ = (mq * inv_bc1) / (sqrtf(v) * inv_sqrt_bc2 + eps);
    }
    tn[r][c] = np_;
    if (d.Np) ((g_f32*)(d.Np))[gr * d.np + gc] = np_;
  }
  if (!d.NpT) return;  // (uniform over the workgroup)
  __syncthreads();
  g_f32* NpT = (g_f32*)(d.NpT);
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;
    NpT[(int64_t(tj) * kTile + r) * d.mp + int64_t(ti) * kTile + c] = tn[c][r];
  }
}

__global__ __launch_bounds__(256) void soap_eye_kernel(const SoapEyeDesc* __restrict__ descs, int count) {
  const int e = find_desc(descs, count, blockIdx.x);
  const SoapEyeDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  const int64_t gc = int64_t(tj) * kTile + c;
  g_f32* X = (g_f32*)(d.X);
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int64_t gr = int64_t(ti) * kTile + rr + 4 * i;
    X[gr * d.ld + gc] = (gr == gc && gr < d.d) ? 1.0f : 0.0f;
  }
}

// Householder factorization of one 16-column panel (LAPACK's convention: for the column x below and
// on the pivot, beta = -sign(x_0) ||x||, tau = (beta - x_0) / beta, v = x / (x_0 - beta) with v_0 = 1;
// tau = 0 when nothing below the pivot is non-zero). Its 16 x 16 block of T receives tau_k on the
// diagonal and the dot products v_j . v_k (j < k) above it, from which the applications and the
// block's factor form what they need. One 512-thread workgroup per panel; thread t holds rows
// t + 512 i (i < 8) of the panel in registers (the panel's columns are rows of the transposed matrix:
// each is read coalesced). One block reduction per column, of 16 sums at once (column k's squared
// norm below the pivot and its products with the other 15 columns there), formed in the same pass
// over the rows that applies the previous reflector; every wave sums the waves' partials itself
// (lane l: slot l, in wave order) and reads them back from its lanes. Every sum is taken in a fixed
// order.
__global__ __launch_bounds__(kQrPanelThreads) void qr_panel_kernel(const QrPanelDesc* __restrict__ descs) {
  __shared__ float red[2][kQrPanelThreads / 64][kQrPanel];  // by column parity: the waves' sums
  __shared__ float piv[2][kQrPanel];                         // by column parity: the pivot row
  __shared__ float Ds[kQrPanel][kQrPanel];
  const QrPanelDesc& d = descs[blockIdx.x];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int jb = d.jb;
  const int rows = jb > 0 ? d.d - d.c : 0;  // panel rows [c, d)
  float a[kQrRowsPerThread][kQrPanel];
  {
    const g_cf32* At = (const g_cf32*)(d.At) + int64_t(d.c) * d.ld + d.c;
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k)
#pragma unroll
      for (int i = 0; i < kQrRowsPerThread; ++i) {
        const int lr = t + kQrPanelThreads * i;
        a[i][k] = (lr < rows && k < jb) ? At[int64_t(k) * d.ld + lr] : 0.0f;
      }
  }
  if (t < kQrPanel * kQrPanel) Ds[t / kQrPanel][t % kQrPanel] = 0.0f;
  // register rows that hold panel rows (uniform); the others are zero and are skipped. Columns
  // >= jb are zero as well: their dot products are exactly 0 and they stay 0.
  const int used = (rows + kQrPanelThreads - 1) / kQrPanelThreads;
  // Column k's sums over the rows below its pivot: slot l = a_k . a_l (slot k: the squared norm),
  // reduced within each wave (lane l: slot l) into red[k & 1]; the pivot row into piv[k & 1].
  auto reduce_col = [&](auto kc) {
    constexpr int k = decltype(kc)::value;
    float part[kQrPanel];
#pragma unroll
    for (int l = 0; l < kQrPanel; ++l) part[l] = 0.0f;
#pragma unroll
    for (int i = 0; i < kQrRowsPerThread; ++i) {
      if (i < used && t + kQrPanelThreads * i > k) {
        const float ak = a[i][k];
#pragma unroll
        for (int l = 0; l < kQrPanel; ++l) part[l] += ak * a[i][l];
      }
    }
    // lane l of every row: the row's sum of slot l; then over the four rows of the wave (the
    // adds are commutative pairs, so every lane of a column l agrees bit for bit)
    const float r = sum_rows4(row_reduce_scatter16(part, lane & 15));
    if (lane < kQrPanel) red[k & 1][w][lane] = r;
    if (t == k) {
#pragma unroll
      for (int l = 0; l < kQrPanel; ++l) piv[k & 1][l] = a[0][l];
    }
  };
  if (jb > 0) {  // (uniform)
    reduce_col(std::integral_constant<int, 0>{});
    __syncthreads();
  }

  // One barrier per column: the sums of column k were formed (and reduced) in the pass that applied
  // reflector k - 1. With them, v_k = e_k + scale a_k (below the pivot), and every product with v_k
  // follows without another reduction: v_k . a_l = a_l[k] + scale (a_k . a_l), v_j . v_k = v_j[k] +
  // scale (a_k . v_j).
  unrolled<kQrPanel>([&](auto kc) {
    constexpr int k = decltype(kc)::value;
    if (k >= jb) return;  // (uniform: jb is the panel's width)
    // the block totals: lane l of every wave sums slot l over the waves in wave order, and the wave
    // reads them from its lanes (red[k & 1] and piv[k & 1] are written again only after the next
    // column's barrier)
    float mine = 0.0f;
#pragma unroll
    for (int j = 0; j < kQrPanelThreads / 64; ++j) mine += red[k & 1][j][lane & (kQrPanel - 1)];
    float tot[kQrPanel], pv[kQrPanel];
#pragma unroll
    for (int l = 0; l < kQrPanel; ++l) {
      tot[l] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mine), l));
      pv[l] = piv[k & 1][l];
    }
    const float alpha = pv[k], sigma = tot[k];
    float tau = 0.0f, scale = 0.0f;
    if (sigma != 0.0f) {
      const float beta = -copysignf(sqrtf(alpha * alpha + sigma), alpha);
      tau = (beta - alpha) / beta;
      scale = 1.0f / (alpha - beta);
    }
    float f[kQrPanel];
#pragma unroll
    for (int l = k + 1; l < kQrPanel; ++l) f[l] = tau * (pv[l] + scale * tot[l]);
#pragma unroll
    for (int i = 0; i < kQrRowsPerThread; ++i) {
      if (i < used) {
        const int lr = t + kQrPanelThreads * i;
        a[i][k] = lr > k ? a[i][k] * scale : (lr == k ? 1.0f : 0.0f);
#pragma unroll
        for (int l = k + 1; l < kQrPanel; ++l) a[i][l] -= f[l] * a[i][k];
      }
    }
#pragma unroll
    for (int j = 0; j < k; ++j)
      if (t == j) Ds[j][k] = pv[j] + scale * tot[j];
    if (t == k) Ds[k][k] = tau;
    if constexpr (k + 1 < kQrPanel) {
      if (k + 1 < jb) {  // (uniform)
        reduce_col(std::integral_constant<int, k + 1>{});
        __syncthreads();
      }
    }
  });
  __syncthreads();
  // the panel's 16 columns of V and rows of Vt over every block row: rows [0, c - j0) above the
  // panel are zero, rows [c - j0, vrows) are the registers (zero from d on; vrows - (c - j0) =
  // dp - c <= kQrMaxDim)
  const int top = d.c - d.j0, s16 = top;  // the panel's first column within the block = c - j0
  {
    g_f32* V = (g_f32*)(d.V) + s16;
    g_f32* Vt = (g_f32*)(d.Vt) + int64_t(s16) * d.ldvt;
    const int below = d.vrows - top;
#pragma unroll
    for (int i = 0; i < kQrRowsPerThread; ++i) {
      const int lr = t + kQrPanelThreads * i;
      if (lr < below) {
        g_f32x4* vrow = (g_f32x4*)(V + int64_t(top + lr) * kQrBlock);
#pragma unroll
        for (int q = 0; q < kQrPanel / 4; ++q)
          vrow[q] = f32x4{a[i][4 * q], a[i][4 * q + 1], a[i][4 * q + 2], a[i][4 * q + 3]};
#pragma unroll
        for (int k = 0; k < kQrPanel; ++k) Vt[int64_t(k) * d.ldvt + top + lr] = a[i][k];
      }
    }
    for (int r = t; r < top; r += kQrPanelThreads) {
#pragma unroll
      for (int q = 0; q < kQrPanel / 4; ++q) ((g_f32x4*)(V + int64_t(r) * kQrBlock))[q] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int k = 0; k < kQrPanel; ++k) Vt[int64_t(k) * d.ldvt + r] = 0.0f;
    }
  }
  if (t < kQrPanel * kQrPanel)
    ((g_f32*)d.T)[int64_t(s16 + t / kQrPanel) * kQrBlock + s16 + t % kQrPanel] = Ds[t / kQrPanel][t % kQrPanel];
}

// x <- H_16 ... H_1 x = x - V_s y for one column x of A (a row of At, rows [c, d) of A), with
// y_k = tau_k (w_k - sum_{j<k} (v_j . v_k) y_j) and w = V_s^T x (the reflectors applied one after the
// other, in the reduced coordinates). Thread t holds entries t + 256 i in registers and forms its
// part of the 16 sums w (the panel's V rows are 64 contiguous bytes); the workgroup reduces them in
// a fixed order (DPP reduce-scatter within each row of 16 lanes, then over the wave's four rows, then
// over the four waves through LDS), one thread runs the 16-step recurrence for y, and every thread
// subtracts V_s y from its entries. The column is read once and written once.
__global__ __launch_bounds__(kQrColThreads) void qr_col_kernel(const QrColDesc* __restrict__ descs, int count) {
  __shared__ float red[kQrColThreads / 64][kQrPanel];
  __shared__ float ws[kQrPanel];
  __shared__ float ys[kQrPanel];
  __shared__ float Ts[kQrPanel][kQrPanel];
  const int e = find_desc(descs, count, blockIdx.x);
  const QrColDesc& d = descs[e];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  static_assert(kQrColThreads == kQrPanel * kQrPanel, "one thread per entry of the panel's block of T");
  Ts[t / kQrPanel][t % kQrPanel] = ((const g_cf32*)(d.T))[(t / kQrPanel) * kQrBlock + t % kQrPanel];
  const int64_t col = int64_t(d.c) + kQrPanel + (blockIdx.x - d.tile_begin);
  g_f32* x = (g_f32*)(d.At) + col * d.ld + d.c;
  const g_cf32* V = (const g_cf32*)(d.V);
  const int used = (d.rows + kQrColThreads - 1) / kQrColThreads;  // uniform
  float xr[kQrColRows];
  float part[kQrPanel];
#pragma unroll
  for (int k = 0; k < kQrPanel; ++k) part[k] = 0.0f;
#pragma unroll
  for (int i = 0; i < kQrColRows; ++i) {
    xr[i] = 0.0f;
    if (i < used) {
      const int r = t + kQrColThreads * i;
      if (r < d.rows) {
        xr[i] = x[r];
        const g_cf32x4* vr = (const g_cf32x4*)(V + int64_t(r) * kQrBlock);
#pragma unroll
        for (int q = 0; q < kQrPanel / 4; ++q) {
          const f32x4 v = vr[q];
#pragma unroll
          for (int j = 0; j < 4; ++j) part[4 * q + j] += v[j] * xr[i];
        }
      }
    }
  }
  const float rsum = sum_rows4(row_reduce_scatter16(part, lane & 15));
  if (lane < kQrPanel) red[w][lane] = rsum;
  __syncthreads();
  if (t < kQrPanel) ws[t] = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
  __syncthreads();
  if (t == 0) {
    float yk[kQrPanel];
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k) {
      float acc = ws[k];
#pragma unroll
      for (int j = 0; j < k; ++j) acc -= Ts[j][k] * yk[j];
      yk[k] = Ts[k][k] * acc;
      ys[k] = yk[k];
    }
  }
  __syncthreads();
  float y[kQrPanel];
#pragma unroll
  for (int k = 0; k < kQrPanel; ++k) y[k] = ys[k];
#pragma unroll
  for (int i = 0; i < kQrColRows; ++i) {
    if (i < used) {
      const int r = t + kQrColThreads * i;
      if (r < d.rows) {
        const g_cf32x4* vr = (const g_cf32x4*)(V + int64_t(r) * kQrBlock);
        float sub = 0.0f;
#pragma unroll
        for (int q = 0; q < kQrPanel / 4; ++q) {
          const f32x4 v = vr[q];
#pragma unroll
          for (int j = 0; j < 4; ++j) sub += v[j] * y[4 * q + j];
        }
        x[r] = xr[i] - sub;
      }
    }
  }
}

// The block's compact-WY factor, held in LDS. Each panel's diagonal block first, row by row (one
// thread per row i; T_kk = tau_k, T_ik = -tau_k sum_{j=i}^{k-1} T_ij (v_j . v_k), from the tau and dot
// products the panel left in its block); then, with the blocks of G above the diagonal blocks (G
// summed over its partials in order), for each panel s = 1 .. 7 (first column n0 = 16 s),
// M = G[0:n0, n0:n0+16] T_s and T[0:n0, n0:n0+16] = -T[0:n0, 0:n0] M over the upper triangle of
// T[0:n0, 0:n0].
__global__ __launch_bounds__(256) void qr_t_kernel(const QrTDesc* __restrict__ descs) {
  __shared__ float Tl[kQrBlock][kQrBlock + 1];
  __shared__ float Gl[kQrBlock][kQrBlock + 1];
  __shared__ float M1[kQrBlock - kQrPanel][kQrPanel + 1];
  __shared__ float Dl[kQrBlock][kQrPanel];  // row i: the panel's tau / dot-product row i
  const QrTDesc& d = descs[blockIdx.x];
  const int t = threadIdx.x;
  g_f32* T = (g_f32*)(d.T);
  const g_cf32* G = (const g_cf32*)(d.G);
  // thread t owns column j = t % 128 and rows i = t / 128 + 2 m (m < 64) of both matrices; the
  // partials of G are summed with every load of one partial in flight together
  constexpr int kM = kQrBlock * kQrBlock / 256;
  const int tj = t % kQrBlock, ti = t / kQrBlock;
  float g[kM];
#pragma unroll
  for (int m = 0; m < kM; ++m) g[m] = 0.0f;
  for (int q = 0; q < d.nG; ++q) {
    const g_cf32* Gq = G + int64_t(q) * kQrBlock * kQrBlock;
#pragma unroll
    for (int m = 0; m < kM; ++m) g[m] += Gq[(ti + 2 * m) * kQrBlock + tj];  // (every partial is whole)
  }
#pragma unroll
  for (int m = 0; m < kM; ++m) {
    const int i = ti + 2 * m;
    Tl[i][tj] = 0.0f;
    Gl[i][tj] = g[m];
  }
  for (int idx = t; idx < kQrBlock * kQrPanel; idx += 256) {
    const int i = idx / kQrPanel, jj = idx % kQrPanel;
    Dl[i][jj] = T[i * kQrBlock + (i / kQrPanel) * kQrPanel + jj];
  }
  __syncthreads();
  if (t < kQrBlock) {
    const int i = t, b0 = (i / kQrPanel) * kQrPanel, ii = i % kQrPanel;
    float row[kQrPanel];
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k) {
      float v = 0.0f;
      if (k == ii) {
        v = Dl[i][ii];
      } else if (k > ii) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < k; ++j)
          if (j >= ii) acc += row[j] * Dl[b0 + j][k];
        v = -Dl[b0 + k][k] * acc;
      }
      row[k] = v;
      Tl[i][b0 + k] = v;
    }
  }
  __syncthreads();
  for (int s = 1; s < kQrBlock / kQrPanel; ++s) {
    const int n0 = kQrPanel * s;
    for (int idx = t; idx < n0 * kQrPanel; idx += 256) {
      const int i = idx / kQrPanel, j = idx % kQrPanel;
      float acc = 0.0f;
#pragma unroll
      for (int k = 0; k < kQrPanel; ++k) acc += Gl[i][n0 + k] * Tl[n0 + k][n0 + j];
      M1[i][j] = acc;
    }
    __syncthreads();
    // T[0:n0, 0:n0] is upper triangular with zeros below (whole 16-row groups summed; four
    // accumulators per group, added in a fixed order)
    for (int idx = t; idx < n0 * kQrPanel; idx += 256) {
      const int i = idx / kQrPanel, j = idx % kQrPanel;
      float acc = 0.0f;
      for (int k0 = (i / kQrPanel) * kQrPanel; k0 < n0; k0 += kQrPanel) {
        float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int k = 0; k < kQrPanel; ++k) p[k & 3] += Tl[i][k0 + k] * M1[k0 + k][j];
        acc += (p[0] + p[1]) + (p[2] + p[3]);
      }
      Tl[i][n0 + j] = -acc;
    }
    __syncthreads();
  }
  for (int idx = t; idx < kQrBlock * kQrBlock; idx += 256) T[idx] = Tl[idx / kQrBlock][idx % kQrBlock];
}

}  // namespace

hipError_t launch_soap_prep(const SoapPrepDesc* d, int count, int total_tiles, float beta1, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(soap_prep_kernel, dim3(total_tiles), dim3(256), 0, st, d, count, beta1);
  return hipGetLastError();
}

hipError_t launch_soap_adam(const SoapAdamDesc* d, int count, int total_tiles, float beta2, float eps,
                            float inv_bc1, float inv_sqrt_bc2, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(soap_adam_kernel, dim3(total_tiles), dim3(256), 0, st, d, count, beta2, eps, inv_bc1,
                     inv_sqrt_bc2);
  return hipGetLastError();
}

hipError_t launch_soap_eye(const SoapEyeDesc* d, int count, int total_tiles, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(soap_eye_kernel, dim3(total_tiles), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_qr_panel(const QrPanelDesc* d, int count, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(qr_panel_kernel, dim3(count), dim3(kQrPanelThreads), 0, st, d);
  return hipGetLastError();
}

hipError_t launch_qr_col(const QrColDesc* d, int count, int total_blocks, hipStream_t st) {
  if (total_blocks <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(qr_col_kernel, dim3(total_blocks), dim3(kQrColThreads), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_qr_t(const QrTDesc* d, int count, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(qr_t_kernel, dim3(count), dim3(256), 0, st, d);
  return hipGetLastError();
}

}  // namespace mfsdp
