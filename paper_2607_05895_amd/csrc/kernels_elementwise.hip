// HBM-bound passes of the owner step: momentum + Nesterov + Frobenius partials (with the NS input
// written in both layouts), the per-matrix norm scale, the parameter update, and AdamW.
// All reductions use a fixed order (no floating-point atomics), so results are deterministic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfsdp_internal.h"

namespace mfsdp {
namespace {

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
  // round to nearest even; NaN stays NaN (quiet bit set)
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

__device__ __forceinline__ float load_as_f32(const void* p, int64_t i, int dt) {
  return dt == kDtBF16 ? bf2f(static_cast<const uint16_t*>(p)[i]) : static_cast<const float*>(p)[i];
}

__device__ __forceinline__ void store_from_f32(void* p, int64_t i, float v, int dt) {
  if (dt == kDtBF16)
    static_cast<uint16_t*>(p)[i] = f2bf(v);
  else
    static_cast<float*>(p)[i] = v;
}

// Store 4 consecutive values (16-byte aligned fp32 or 8-byte aligned bf16 destination).
template <int DT>
__device__ __forceinline__ void store4(void* base, int64_t idx, const float v[4]) {
  if constexpr (DT == kDtBF16) {
    uint2 w;
    w.x = uint32_t(f2bf(v[0])) | (uint32_t(f2bf(v[1])) << 16);
    w.y = uint32_t(f2bf(v[2])) | (uint32_t(f2bf(v[3])) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(base) + idx) = w;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(base) + idx) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <int DT>
__device__ __forceinline__ void load4(const void* base, int64_t idx, float v[4]) {
  if constexpr (DT == kDtBF16) {
    uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(base) + idx);
    v[0] = __uint_as_float(w.x << 16);
    v[1] = __uint_as_float(w.x & 0xffff0000u);
    v[2] = __uint_as_float(w.y << 16);
    v[3] = __uint_as_float(w.y & 0xffff0000u);
  } else {
    float4 f = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + idx);
    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
  }
}

// Entry lookup: the largest i with begin(i) <= key (begins are increasing, begin(0) = 0).
template <typename D>
__device__ __forceinline__ int find_entry(const D* descs, int count, int key) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (descs[mid].tile_begin <= key) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ---------------------------------------------------------------------------------------------
// prep: one 64 x 64 tile of the stored (padded) matrix per workgroup of 256 threads.
// Thread t owns columns 4*(t%16) .. +3 of rows t/16 + 16 q, q = 0..3.
template <int NSDT>
__global__ __launch_bounds__(256) void prep_kernel(const PrepDesc* __restrict__ descs, int count,
                                                   float beta, float omb, int nesterov) {
  __shared__ float tile[64][65];
  __shared__ float red[4];
  const int e = find_entry(descs, count, blockIdx.x);
  const PrepDesc d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int64_t row0 = int64_t(lt / d.tiles_n) * 64, col0 = int64_t(lt % d.tiles_n) * 64;
  const int t = threadIdx.x;
  const int c4 = (t & 15) * 4, rr = t >> 4;
  float ss = 0.0f;
  const bool vec = (d.n % 4 == 0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t i = row0 + rr + 16 * q;
    const int64_t j0 = col0 + c4;
    float u[4];
    if (i < d.m && vec && j0 + 3 < d.n) {
      const int64_t idx = i * d.n + j0;
      float g[4];
      if (d.grad_dtype == kDtBF16) load4<kDtBF16>(d.grad, idx, g); else load4<kDtF32>(d.grad, idx, g);
      if (d.momentum) {
        float4 mo = *reinterpret_cast<const float4*>(d.momentum + idx);
        float mv[4] = {mo.x, mo.y, mo.z, mo.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          mv[k] = mv[k] + omb * (g[k] - mv[k]);
          u[k] = nesterov ? g[k] + beta * (mv[k] - g[k]) : mv[k];
        }
        *reinterpret_cast<float4*>(d.momentum + idx) = make_float4(mv[0], mv[1], mv[2], mv[3]);
      } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) u[k] = g[k];
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t j = j0 + k;
        u[k] = 0.0f;
        if (i < d.m && j < d.n) {
          const int64_t idx = i * d.n + j;
          const float g = load_as_f32(d.grad, idx, d.grad_dtype);
          if (d.momentum) {
            float mv = d.momentum[idx];
            mv = mv + omb * (g - mv);
            d.momentum[idx] = mv;
            u[k] = nesterov ? g + beta * (mv - g) : mv;
          } else {
            u[k] = g;
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      ss += u[k] * u[k];
      tile[rr + 16 * q][c4 + k] = u[k];
    }
    store4<NSDT>(d.d_out, i * d.ld_d + j0, u);
  }
  __syncthreads();
  // transposed copy: rows col0 + jj of the T buffer, columns row0 + c4 .. +3
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int jj = rr + 16 * q;
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = tile[c4 + k][jj];
    store4<NSDT>(d.t_out, (col0 + jj) * d.ld_t + row0 + c4, v);
  }
  ss = wave_sum(ss);
  if ((t & 63) == 0) red[t >> 6] = ss;
  __syncthreads();
  if (t == 0) d.partials[lt] = (red[0] + red[1]) + (red[2] + red[3]);
}

// ---------------------------------------------------------------------------------------------
// norm: one workgroup per matrix; fixed-order sum of the tile partials in fp64.
__global__ __launch_bounds__(256) void norm_kernel(const NormDesc* __restrict__ descs, float eps) {
  __shared__ double red[256];
  const NormDesc d = descs[blockIdx.x];
  double s = 0.0;
  for (int i = threadIdx.x; i < d.count; i += 256) s += double(d.partials[i]);
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double nrm = sqrt(red[0]);
    d.scale[0] = float(1.0 / (nrm > double(eps) ? nrm : double(eps)));
  }
}

// ---------------------------------------------------------------------------------------------
// apply: one 64 x 64 tile of the stored m x n matrix per workgroup (no padding here).
template <int NSDT>
__global__ __launch_bounds__(256) void apply_kernel(const ApplyDesc* __restrict__ descs, int count) {
  const int e = find_entry(descs, count, blockIdx.x);
  const ApplyDesc d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int64_t row0 = int64_t(lt / d.tiles_n) * 64, col0 = int64_t(lt % d.tiles_n) * 64;
  const int t = threadIdx.x;
  const int c4 = (t & 15) * 4, rr = t >> 4;
  const float osc = d.use_scale ? d.scale[0] : 1.0f;
  const bool vec = (d.n % 4 == 0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t i = row0 + rr + 16 * q;
    if (i >= d.m) continue;
    const int64_t j0 = col0 + c4;
    float o[4];
    load4<NSDT>(d.o, i * d.ld_o + j0, o);  // the padded O buffer always has the 4 columns
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] *= osc;
    const int64_t idx = i * d.n + j0;
    if (vec && j0 + 3 < d.n) {
      if (d.mode == 0) {
        float p[4];
        if (d.param_dtype == kDtBF16) load4<kDtBF16>(d.param, idx, p); else load4<kDtF32>(d.param, idx, p);
#pragma unroll
        for (int k = 0; k < 4; ++k) p[k] = p[k] * d.decay - d.step * o[k];
        if (d.param_dtype == kDtBF16) store4<kDtBF16>(d.param, idx, p); else store4<kDtF32>(d.param, idx, p);
        if (d.update_out) store4<kDtF32>(d.update_out, idx, o);
      } else {
        if (d.param_dtype == kDtBF16) store4<kDtBF16>(d.param, idx, o); else store4<kDtF32>(d.param, idx, o);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (j0 + k >= d.n) break;
        if (d.mode == 0) {
          const float p = load_as_f32(d.param, idx + k, d.param_dtype);
          store_from_f32(d.param, idx + k, p * d.decay - d.step * o[k], d.param_dtype);
          if (d.update_out) d.update_out[idx + k] = o[k];
        } else {
          store_from_f32(d.param, idx + k, o[k], d.param_dtype);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// AdamW: grouped over up to kAdamWMaxPerLaunch tensors passed by value; each workgroup owns
// kAdamWBlockElems consecutive elements of one tensor, 16 per thread (4 groups of 4).
__device__ __forceinline__ void adamw_elem(float& p, float g, float& m, float& v, const AdamWBatch& b) {
  p = p * b.decay;
  m = m + b.omb1 * (g - m);
  v = b.beta2 * v + b.omb2 * g * g;
  const float denom = sqrtf(v) * b.inv_sqrt_bc2 + b.eps;
  p = p - b.step_size * (m / denom);
}

__global__ __launch_bounds__(256) void adamw_kernel(const AdamWBatch batch) {
  int e = 0;
  for (int k = 1; k < batch.count; ++k)
    if (batch.d[k].block_begin <= int(blockIdx.x)) e = k;
  const AdamWDesc& d = batch.d[e];
  const int64_t base = int64_t(blockIdx.x - d.block_begin) * kAdamWBlockElems;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t i0 = base + (int64_t(q) * 256 + threadIdx.x) * 4;
    if (i0 >= d.numel) break;
    if (i0 + 3 < d.numel) {
      float p[4], g[4];
      if (d.param_dtype == kDtBF16) load4<kDtBF16>(d.param, i0, p); else load4<kDtF32>(d.param, i0, p);
      if (d.grad_dtype == kDtBF16) load4<kDtBF16>(d.grad, i0, g); else load4<kDtF32>(d.grad, i0, g);
      float4 m4 = *reinterpret_cast<const float4*>(d.exp_avg + i0);
      float4 v4 = *reinterpret_cast<const float4*>(d.exp_avg_sq + i0);
      float m[4] = {m4.x, m4.y, m4.z, m4.w}, v[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
      for (int k = 0; k < 4; ++k) adamw_elem(p[k], g[k], m[k], v[k], batch);
      if (d.param_dtype == kDtBF16) store4<kDtBF16>(d.param, i0, p); else store4<kDtF32>(d.param, i0, p);
      *reinterpret_cast<float4*>(d.exp_avg + i0) = make_float4(m[0], m[1], m[2], m[3]);
      *reinterpret_cast<float4*>(d.exp_avg_sq + i0) = make_float4(v[0], v[1], v[2], v[3]);
    } else {
      for (int64_t i = i0; i < d.numel; ++i) {
        float p = load_as_f32(d.param, i, d.param_dtype);
        const float g = load_as_f32(d.grad, i, d.grad_dtype);
        float m = d.exp_avg[i], v = d.exp_avg_sq[i];
        adamw_elem(p, g, m, v, batch);
        store_from_f32(d.param, i, p, d.param_dtype);
        d.exp_avg[i] = m;
        d.exp_avg_sq[i] = v;
      }
    }
  }
}

}  // namespace

hipError_t launch_prep(const PrepDesc* d_descs, int count, int total_tiles, int ns_dtype,
                       float beta, float one_minus_beta, int nesterov, hipStream_t st) {
  if (total_tiles <= 0) return hipSuccess;
  if (ns_dtype == kDtBF16)
    hipLaunchKernelGGL(prep_kernel<kDtBF16>, dim3(total_tiles), dim3(256), 0, st, d_descs, count,
                       beta, one_minus_beta, nesterov);
  else
    hipLaunchKernelGGL(prep_kernel<kDtF32>, dim3(total_tiles), dim3(256), 0, st, d_descs, count,
                       beta, one_minus_beta, nesterov);
  return hipGetLastError();
}

hipError_t launch_norm(const NormDesc* d_descs, int count, float eps, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(norm_kernel, dim3(count), dim3(256), 0, st, d_descs, eps);
  return hipGetLastError();
}

hipError_t launch_apply(const ApplyDesc* d_descs, int count, int total_tiles, int ns_dtype,
                        hipStream_t st) {
  if (total_tiles <= 0) return hipSuccess;
  if (ns_dtype == kDtBF16)
    hipLaunchKernelGGL(apply_kernel<kDtBF16>, dim3(total_tiles), dim3(256), 0, st, d_descs, count);
  else
    hipLaunchKernelGGL(apply_kernel<kDtF32>, dim3(total_tiles), dim3(256), 0, st, d_descs, count);
  return hipGetLastError();
}

hipError_t launch_adamw(const AdamWBatch& batch, int total_blocks, hipStream_t st) {
  if (total_blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(adamw_kernel, dim3(total_blocks), dim3(256), 0, st, batch);
  return hipGetLastError();
}

}  // namespace mfsdp
