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
  g_f32* Gp = (g_f32*)(d.Gp);
  g_f32* GMt = (g_f32*)(d.GMt);
  g_f32* GM = (g_f32*)(d.GM);
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
    if (Gp) Gp[gr * d.np + gc] = g;
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
    GMt[o] = tg[c][r];
    GMt[o + d.np * d.mp] = tm[c][r];
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
  if (gc >= d.d) return;
  g_f32* X = (g_f32*)(d.X);
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int64_t gr = int64_t(ti) * kTile + rr + 4 * i;
    if (gr < d.d) X[gr * d.ld + gc] = gr == gc ? 1.0f : 0.0f;
  }
}

// Householder factorization of one 16-column panel (LAPACK's convention: for the column x below and
// on the pivot, beta = -sign(x_0) ||x||, tau = (beta - x_0) / beta, v = x / (x_0 - beta) with v_0 = 1;
// tau = 0 when nothing below the pivot is non-zero) and the compact-WY factor T of the panel
// (T_kk = tau_k, T_{0:k,k} = -tau_k T_{0:k,0:k} V_{:,0:k}^T v_k), so that H_1 ... H_jb = I - V T V^T.
// One 512-thread workgroup per panel; thread t holds rows t + 512 i (i < 8) of the panel in
// registers. Per column: one block reduction for the norm below the pivot, one for the 15 dot
// products v_k . a_l (l > k, to update the later columns) and v_i . v_k (i < k, for T), whose 15
// totals are formed once in LDS and then read by every thread. Every sum is
// taken in a fixed order.
__global__ __launch_bounds__(kQrPanelThreads) void qr_panel_kernel(const QrPanelDesc* __restrict__ descs) {
  __shared__ float red1[kQrPanelThreads / 64];
  __shared__ float red2[kQrPanelThreads / 64][kQrPanel];
  __shared__ float tot[kQrPanel];
  __shared__ float alpha_s;
  __shared__ float Ts[kQrPanel][kQrPanel];
  const QrPanelDesc& d = descs[blockIdx.x];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int jb = d.jb;
  float a[kQrRowsPerThread][kQrPanel];
#pragma unroll
  for (int i = 0; i < kQrRowsPerThread; ++i) {
    const int lr = t + kQrPanelThreads * i;
    if (lr < d.rows) {
      const g_cf32x4* row = (const g_cf32x4*)(d.A + (int64_t(d.j0) + lr) * d.lda + d.j0);
#pragma unroll
      for (int q = 0; q < kQrPanel / 4; ++q) {
        const f32x4 v = row[q];
#pragma unroll
        for (int j = 0; j < 4; ++j) a[i][4 * q + j] = (4 * q + j < jb) ? v[j] : 0.0f;
      }
    } else {
#pragma unroll
      for (int k = 0; k < kQrPanel; ++k) a[i][k] = 0.0f;
    }
  }
  if (t < kQrPanel * kQrPanel) Ts[t / kQrPanel][t % kQrPanel] = 0.0f;
  // register rows that hold panel rows (uniform); the others are zero and are skipped. Columns
  // >= jb are zero as well: their dot products are exactly 0 and they stay 0.
  const int used = (d.rows + kQrPanelThreads - 1) / kQrPanelThreads;

  unrolled<kQrPanel>([&](auto kc) {
    constexpr int k = decltype(kc)::value;
    if (k >= jb) return;  // (uniform: jb is the panel's width)
    // norm of the column below the pivot (local row k), and the pivot itself
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < kQrRowsPerThread; ++i) {
      const int lr = t + kQrPanelThreads * i;
      if (i < used && lr > k) s += a[i][k] * a[i][k];
    }
    s = wave_sum(s);
    if (lane == 0) red1[w] = s;
    if (t == k) alpha_s = a[0][k];
    __syncthreads();
    float sigma = 0.0f;
#pragma unroll
    for (int j = 0; j < kQrPanelThreads / 64; ++j) sigma += red1[j];
    const float alpha = alpha_s;
    float tau = 0.0f, scale = 0.0f;
    if (sigma != 0.0f) {
      const float beta = -copysignf(sqrtf(alpha * alpha + sigma), alpha);
      tau = (beta - alpha) / beta;
      scale = 1.0f / (alpha - beta);
    }
#pragma unroll
    for (int i = 0; i < kQrRowsPerThread; ++i) {
      if (i < used) {
        const int lr = t + kQrPanelThreads * i;
        a[i][k] = lr > k ? a[i][k] * scale : (lr == k ? 1.0f : 0.0f);
      }
    }
    // slot s < k: v_s . v_k (for T); slot s >= k: v_k . a_{s+1} (to update column s + 1)
    {
      float part[kQrPanel];
#pragma unroll
      for (int sl = 0; sl < kQrPanel; ++sl) part[sl] = 0.0f;
#pragma unroll
      for (int i = 0; i < kQrRowsPerThread; ++i) {
        if (i < used) {
          const float vk = a[i][k];
#pragma unroll
          for (int sl = 0; sl < kQrPanel - 1; ++sl) part[sl] += vk * a[i][sl < k ? sl : sl + 1];
        }
      }
      // lane l of every row: the row's sum of slot l; then over the four rows of the wave (the
      // adds are commutative pairs, so every lane of a column l agrees bit for bit)
      float r = row_reduce_scatter16(part, lane & 15);
      r += __shfl_xor(r, 16);
      r += __shfl_xor(r, 32);
      if (lane < kQrPanel - 1) red2[w][lane] = r;
    }
    __syncthreads();
    // the 15 block totals, each summed once over the waves in wave order
    if (t < kQrPanel - 1) {
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < kQrPanelThreads / 64; ++j) acc += red2[j][t];
      tot[t] = acc;
    }
    __syncthreads();
    auto total = [&](int sl) { return tot[sl]; };
    float f[kQrPanel];
#pragma unroll
    for (int l = k + 1; l < kQrPanel; ++l) f[l] = tau * total(l - 1);
#pragma unroll
    for (int i = 0; i < kQrRowsPerThread; ++i) {
      if (i < used) {
#pragma unroll
        for (int l = k + 1; l < kQrPanel; ++l) a[i][l] -= f[l] * a[i][k];
      }
    }
    if (t < k) {
      float acc = 0.0f;
#pragma unroll
      for (int j = 0; j < k; ++j)
        if (j >= t) acc += Ts[t][j] * total(j);
      Ts[t][k] = -tau * acc;
    } else if (t == k) {
      Ts[k][k] = tau;
    }
  });
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kQrRowsPerThread; ++i) {
    const int lr = t + kQrPanelThreads * i;
    if (lr < d.rows) {
      g_f32x4* vrow = (g_f32x4*)(d.V + int64_t(lr) * kQrPanel);
#pragma unroll
      for (int q = 0; q < kQrPanel / 4; ++q)
        vrow[q] = f32x4{a[i][4 * q], a[i][4 * q + 1], a[i][4 * q + 2], a[i][4 * q + 3]};
    }
  }
  if (t < kQrPanel * kQrPanel) ((g_f32*)d.T)[t] = Ts[t / kQrPanel][t % kQrPanel];
}

// X <- X - V (T^T (V^T X)) on one block of 64 columns, all `rows` rows. Thread (q, g) = (t % 16,
// t / 16) owns the column quad 4q .. 4q + 3 and the rows g, g + 16, ... (16-byte loads and stores).
// A first pass forms the 16 column sums W = V^T X: per thread, then over the four row groups of a
// wave (lanes 16 and 32 apart), then over the four waves through LDS, in a fixed order; one wave
// forms Y = T^T W; a second pass subtracts V Y.
__global__ __launch_bounds__(256) void qr_apply_kernel(const QrApplyDesc* __restrict__ descs, int count) {
  __shared__ float red[4][kQrPanel][kQrApplyCols];
  __shared__ float ys[kQrPanel][kQrApplyCols];
  const int e = find_desc(descs, count, blockIdx.x);
  const QrApplyDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int q = t & 15, g = t >> 4;
  const int lc = lt * kQrApplyCols + 4 * q;  // first column of this thread's quad, within [0, cols)
  const bool live = lc < d.cols, full = lc + 4 <= d.cols;
  g_f32* X = (g_f32*)(d.X) + int64_t(d.row0) * d.ldx + d.c0 + (live ? lc : 0);
  const g_cf32x4* V = (const g_cf32x4*)(d.V);
  auto load4 = [&](int64_t o) -> f32x4 {
    if (full) return *(const g_cf32x4*)(X + o);
    f32x4 x = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lc + j < d.cols) x[j] = X[o + j];
    return x;
  };
  float wk[4][kQrPanel];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k) wk[j][k] = 0.0f;
  if (live) {
#pragma unroll 4
    for (int r = g; r < d.rows; r += 16) {
      const f32x4 x = load4(int64_t(r) * d.ldx);
#pragma unroll
      for (int qq = 0; qq < kQrPanel / 4; ++qq) {
        const f32x4 v = V[int64_t(r) * (kQrPanel / 4) + qq];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) wk[j][4 * qq + i] += v[i] * x[j];
      }
    }
  }
  // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same columns (row groups 4w .. 4w + 3)
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k) {
      float v = wk[j][k];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      wk[j][k] = v;
    }
  if (lane < 16) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int k = 0; k < kQrPanel; ++k) red[w][k][4 * q + j] = wk[j][k];
  }
  __syncthreads();
  if (t < kQrApplyCols) {
    const g_cf32* T = (const g_cf32*)(d.T);
    float W[kQrPanel];
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k) W[k] = ((red[0][k][t] + red[1][k][t]) + red[2][k][t]) + red[3][k][t];
#pragma unroll
    for (int i = 0; i < kQrPanel; ++i) {
      float y = 0.0f;
#pragma unroll
      for (int k = 0; k <= i; ++k) y += T[k * kQrPanel + i] * W[k];
      ys[i][t] = y;
    }
  }
  __syncthreads();
  if (!live) return;
  float y[4][kQrPanel];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int k = 0; k < kQrPanel; ++k) y[j][k] = ys[k][4 * q + j];
#pragma unroll 4
  for (int r = g; r < d.rows; r += 16) {
    const int64_t o = int64_t(r) * d.ldx;
    f32x4 x = load4(o);
    f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int qq = 0; qq < kQrPanel / 4; ++qq) {
      const f32x4 v = V[int64_t(r) * (kQrPanel / 4) + qq];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) s[j] += v[i] * y[j][4 * qq + i];
    }
    if (full) {
      *(g_f32x4*)(X + o) = x - s;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (lc + j < d.cols) X[o + j] = x[j] - s[j];
    }
  }
}

// Transposed boundary copy: dst[c][r] = src[r][c] for r < rows, c < cols (64 x 64 tiles over the
// real block, through a padded LDS tile).
__global__ __launch_bounds__(256) void copy_out_t_kernel(const ShCopyDesc* __restrict__ descs, int count) {
  __shared__ float tt[kTile][kTile + 1];
  const int e = find_desc(descs, count, blockIdx.x);
  const ShCopyDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  const g_cf32* src = (const g_cf32*)(d.src);
  g_f32* dst = (g_f32*)(d.dst);
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;
    const int64_t gr = int64_t(ti) * kTile + r, gc = int64_t(tj) * kTile + c;
    tt[r][c] = (gr < d.rows && gc < d.cols) ? src[gr * d.ld_src + gc] : 0.0f;
  }
  __syncthreads();
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;  // destination row = source column
    const int64_t dr = int64_t(tj) * kTile + r, dc = int64_t(ti) * kTile + c;
    if (dr < d.cols && dc < d.rows) dst[dr * d.ld_dst + dc] = tt[c][r];
  }
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

hipError_t launch_qr_apply(const QrApplyDesc* d, int count, int total_blocks, hipStream_t st) {
  if (total_blocks <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(qr_apply_kernel, dim3(total_blocks), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_copy_out_transposed(const ShCopyDesc* d, int count, int total_tiles, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_out_t_kernel, dim3(total_tiles), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

}  // namespace mfsdp
