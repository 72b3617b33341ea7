// HBM-bound passes of the owner step: momentum + Nesterov + Frobenius partials (with the NS input
// written in both layouts), the per-matrix norm scale, the parameter update, and AdamW.
// All reductions use a fixed order (no floating-point atomics), so results are deterministic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "mfsdp_internal.h"

namespace mfsdp {
namespace {

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) { return uint16_t(pack_bf16x2(f, 0.0f)); }

__device__ __forceinline__ float load_as_f32(const void* p, int64_t i, int dt) {
  return dt == kDtBF16 ? bf2f(static_cast<const uint16_t*>(p)[i]) : static_cast<const float*>(p)[i];
}

__device__ __forceinline__ void store_from_f32(void* p, int64_t i, float v, int dt) {
  if (dt == kDtBF16)
    static_cast<uint16_t*>(p)[i] = f2bf(v);
  else
    static_cast<float*>(p)[i] = v;
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
// 8-element vector helpers (16 B of bf16, 32 B of fp32). NT = non-temporal access (measured to
// help the parameter-update pass and to hurt the momentum pass).
struct V8 { float v[8]; };

// Every buffer here is device memory; accessing it through global-address-space pointers gives
// global_load/global_store instead of flat instructions (which also count against lgkmcnt).
template <typename V>
using gptr = __attribute__((address_space(1))) V*;

template <bool NT, typename V>
__device__ __forceinline__ V ld_stream(const V* p) {
  const gptr<const V> g = (gptr<const V>)p;
  if constexpr (NT) return __builtin_nontemporal_load(g);
  else return *g;
}
template <bool NT, typename V>
__device__ __forceinline__ void st_stream(V* p, V v) {
  const gptr<V> g = (gptr<V>)p;
  if constexpr (NT) __builtin_nontemporal_store(v, g);
  else *g = v;
}

template <int DT, bool NT = false>
__device__ __forceinline__ void load8(const void* base, int64_t idx, V8& x) {
  if constexpr (DT == kDtBF16) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 w = ld_stream<NT>(reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(base) + idx));
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x.v[2 * k] = __uint_as_float(u[k] << 16);
      x.v[2 * k + 1] = __uint_as_float(u[k] & 0xffff0000u);
    }
  } else {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 a = ld_stream<NT>(reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + idx));
    const f32x4 b = ld_stream<NT>(reinterpret_cast<const f32x4*>(static_cast<const float*>(base) + idx + 4));
    x.v[0] = a.x; x.v[1] = a.y; x.v[2] = a.z; x.v[3] = a.w;
    x.v[4] = b.x; x.v[5] = b.y; x.v[6] = b.z; x.v[7] = b.w;
  }
}

template <int DT, bool NT = false>
__device__ __forceinline__ void store8(void* base, int64_t idx, const V8& x) {
  if constexpr (DT == kDtBF16) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 w;
    w.x = pack_bf16x2(x.v[0], x.v[1]);
    w.y = pack_bf16x2(x.v[2], x.v[3]);
    w.z = pack_bf16x2(x.v[4], x.v[5]);
    w.w = pack_bf16x2(x.v[6], x.v[7]);
    st_stream<NT>(reinterpret_cast<u32x4*>(static_cast<uint16_t*>(base) + idx), w);
  } else {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    float* p = static_cast<float*>(base) + idx;
    st_stream<NT>(reinterpret_cast<f32x4*>(p), f32x4{x.v[0], x.v[1], x.v[2], x.v[3]});
    st_stream<NT>(reinterpret_cast<f32x4*>(p + 4), f32x4{x.v[4], x.v[5], x.v[6], x.v[7]});
  }
}

// ---------------------------------------------------------------------------------------------
// prep: one tile of 64 rows x TW columns of the stored (padded) matrix per workgroup of 256
// threads (TW = kPrepColsBF16 on the bf16 path, 64 on the fp32 path). Phase 1: thread t owns columns
// 8 (t % (TW/8)) .. +7 of rows t / (TW/8) + (2048/TW) q: gradient and momentum in 16-B vectors,
// u to the stored-orientation buffer and to an LDS tile. Phase 2: the transposed copy; thread t
// gathers 8 consecutive tile rows 8 (t % 8) .. +7 of tile column t / 8 + 32 q and writes them as one
// 16-B (bf16) vector, so 8 lanes cover 128 contiguous bytes of a transposed row. In LDS, element
// (i, j) sits at column j ^ 8 ((i >> 3) & 7): the 16-B row writes stay contiguous and the 8-row
// column gathers of a wave hit distinct banks.
// Non-temporal stores of the NS input u and u^T (they are read back from HBM by the first NS
// products anyway: the iterate does not fit the caches at the sizes that matter).
constexpr bool kPrepNtU = true;

template <int NSDT>
struct PrepTraits {
  using elem = typename std::conditional<NSDT == kDtBF16, uint16_t, float>::type;
  static constexpr int TW = NSDT == kDtBF16 ? kPrepColsBF16 : kPrepColsF32;
};

// RED: the entries' gradients are reductions of gradient parts (a separate instantiation keeps the
// plain momentum pass at its register count).
template <int NSDT, bool RED>
__global__ __launch_bounds__(256) void prep_kernel(const PrepDesc* __restrict__ descs, int count,
                                                   float beta, float omb, int nesterov) {
  using T = typename PrepTraits<NSDT>::elem;
  constexpr int TW = PrepTraits<NSDT>::TW;
  constexpr int CPR = TW / 8;          // 8-column chunks per tile row
  constexpr int RPP = 256 / CPR;       // tile rows covered per pass
  __shared__ __attribute__((aligned(16))) T tile[64 * TW];
  __shared__ float red[4];
  const int e = find_entry(descs, count, blockIdx.x);
  const PrepDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int64_t row0 = int64_t(lt / d.tiles_n) * 64, col0 = int64_t(lt % d.tiles_n) * TW;
  const int64_t m = d.m, n = d.n;
  const int t = threadIdx.x;
  const int c8 = (t % CPR) * 8, rr = t / CPR;
  float ss = 0.0f;
  const bool vec = (n % 8 == 0);
  constexpr int NP = 64 / RPP;         // passes over the tile rows
  // u of pass q: to the stored-orientation buffer and to the LDS tile
  auto emit = [&](int q, const V8& u) {
    const int ti = rr + RPP * q;
    const int64_t i = row0 + ti;
    const int64_t j0 = col0 + c8;
#pragma unroll
    for (int k = 0; k < 8; ++k) ss += u.v[k] * u.v[k];
    store8<NSDT, kPrepNtU>(d.d_out, blk_index(i, j0, d.ld_d), u);
    // LDS copy (rounded to the NS dtype exactly as the global one)
    T* trow = tile + ti * TW + (c8 ^ (8 * ((ti >> 3) & 7)));
    if constexpr (NSDT == kDtBF16) {
      uint4 w;
      w.x = pack_bf16x2(u.v[0], u.v[1]);
      w.y = pack_bf16x2(u.v[2], u.v[3]);
      w.z = pack_bf16x2(u.v[4], u.v[5]);
      w.w = pack_bf16x2(u.v[6], u.v[7]);
      *reinterpret_cast<uint4*>(trow) = w;
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) trow[k] = u.v[k];
    }
  };
  if (vec && row0 + 64 <= m && col0 + TW <= n) {
    // interior tile: every load of the tile is issued before the first result is formed
    auto interior = [&](auto gdt) {
      constexpr int GDT = decltype(gdt)::value;
      V8 g[NP], mv[NP];
      if constexpr (!RED) {
#pragma unroll
        for (int q = 0; q < NP; ++q) load8<GDT>(d.grad, (row0 + rr + RPP * q) * n + col0 + c8, g[q]);
      } else {
        // owner-side reduction of the shard span's contributions, in part order
#pragma unroll
        for (int q = 0; q < NP; ++q) load8<GDT>(d.parts[0], (row0 + rr + RPP * q) * n + col0 + c8, g[q]);
        for (int w = 1; w < d.nparts; ++w) {
          const void* pw = d.parts[w];
          V8 t[NP];
#pragma unroll
          for (int q = 0; q < NP; ++q) load8<GDT>(pw, (row0 + rr + RPP * q) * n + col0 + c8, t[q]);
#pragma unroll
          for (int q = 0; q < NP; ++q)
#pragma unroll
            for (int k = 0; k < 8; ++k) g[q].v[k] += t[q].v[k];
        }
#pragma unroll
        for (int q = 0; q < NP; ++q) {
#pragma unroll
          for (int k = 0; k < 8; ++k) g[q].v[k] *= d.gscale;
          if (d.gout) store8<GDT>(d.gout, (row0 + rr + RPP * q) * n + col0 + c8, g[q]);
        }
      }
      if (d.momentum) {
#pragma unroll
        for (int q = 0; q < NP; ++q) load8<kDtF32>(d.momentum, (row0 + rr + RPP * q) * n + col0 + c8, mv[q]);
#pragma unroll
        for (int q = 0; q < NP; ++q) {
          V8 u;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            mv[q].v[k] = mv[q].v[k] + omb * (g[q].v[k] - mv[q].v[k]);
            u.v[k] = nesterov ? g[q].v[k] + beta * (mv[q].v[k] - g[q].v[k]) : mv[q].v[k];
          }
          store8<kDtF32>(d.momentum, (row0 + rr + RPP * q) * n + col0 + c8, mv[q]);
          emit(q, u);
        }
      } else {
#pragma unroll
        for (int q = 0; q < NP; ++q) emit(q, g[q]);
      }
    };
    if (d.grad_dtype == kDtBF16) interior(std::integral_constant<int, kDtBF16>{});
    else interior(std::integral_constant<int, kDtF32>{});
  } else {
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      const int64_t i = row0 + rr + RPP * q;
      const int64_t j0 = col0 + c8;
      V8 u;
      if (i < m && vec && j0 + 7 < n) {
        const int64_t idx = i * n + j0;
        V8 g;
        if constexpr (!RED) {
          if (d.grad_dtype == kDtBF16) load8<kDtBF16>(d.grad, idx, g); else load8<kDtF32>(d.grad, idx, g);
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k) g.v[k] = 0.0f;
          for (int w = 0; w < d.nparts; ++w) {
            V8 t;
            if (d.grad_dtype == kDtBF16) load8<kDtBF16>(d.parts[w], idx, t); else load8<kDtF32>(d.parts[w], idx, t);
#pragma unroll
            for (int k = 0; k < 8; ++k) g.v[k] = w == 0 ? t.v[k] : g.v[k] + t.v[k];
          }
#pragma unroll
          for (int k = 0; k < 8; ++k) g.v[k] *= d.gscale;
          if (d.gout) {
            if (d.grad_dtype == kDtBF16) store8<kDtBF16>(d.gout, idx, g); else store8<kDtF32>(d.gout, idx, g);
          }
        }
        if (d.momentum) {
          V8 mv;
          load8<kDtF32>(d.momentum, idx, mv);
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            mv.v[k] = mv.v[k] + omb * (g.v[k] - mv.v[k]);
            u.v[k] = nesterov ? g.v[k] + beta * (mv.v[k] - g.v[k]) : mv.v[k];
          }
          store8<kDtF32>(d.momentum, idx, mv);
        } else {
          u = g;
        }
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int64_t j = j0 + k;
          u.v[k] = 0.0f;
          if (i < m && j < n) {
            const int64_t idx = i * n + j;
            float g;
            if constexpr (!RED) {
              g = load_as_f32(d.grad, idx, d.grad_dtype);
            } else {
              g = load_as_f32(d.parts[0], idx, d.grad_dtype);
              for (int w = 1; w < d.nparts; ++w) g += load_as_f32(d.parts[w], idx, d.grad_dtype);
              g *= d.gscale;
              if (d.gout) store_from_f32(d.gout, idx, g, d.grad_dtype);
            }
            if (d.momentum) {
              float mv = d.momentum[idx];
              mv = mv + omb * (g - mv);
              d.momentum[idx] = mv;
              u.v[k] = nesterov ? g + beta * (mv - g) : mv;
            } else {
              u.v[k] = g;
            }
          }
        }
      }
      emit(q, u);
    }
  }
  __syncthreads();
  // transposed copy: buffer row col0 + jj, columns row0 + 8 mm .. +7
  {
    const int mm = t & 7;
#pragma unroll
    for (int q = 0; q < TW / 32; ++q) {
      const int jj = (t >> 3) + 32 * q;
      T* dst = static_cast<T*>(d.t_out) + blk_index(col0 + jj, row0 + 8 * mm, d.ld_t);
      if constexpr (NSDT == kDtBF16) {
        uint32_t h[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int ti = 8 * mm + k;
          h[k] = tile[ti * TW + (jj ^ (8 * ((ti >> 3) & 7)))];
        }
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        st_stream<kPrepNtU>(reinterpret_cast<u32x4*>(dst),
                            u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)});
      } else {
        float v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int ti = 8 * mm + k;
          v[k] = tile[ti * TW + (jj ^ (8 * ((ti >> 3) & 7)))];
        }
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        st_stream<kPrepNtU>(reinterpret_cast<f32x4*>(dst), f32x4{v[0], v[1], v[2], v[3]});
        st_stream<kPrepNtU>(reinterpret_cast<f32x4*>(dst + 4), f32x4{v[4], v[5], v[6], v[7]});
      }
    }
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
// apply: one kApplyRows x kApplyCols tile of the stored m x n matrix per workgroup (no padding
// here); thread t owns columns 8 (t % (kApplyCols / 8)) .. +7 of rows t / (kApplyCols / 8) + ...,
// in 16-B vectors.
template <int NSDT>
__global__ __launch_bounds__(256) void apply_kernel(const ApplyDesc* __restrict__ descs, int count) {
  const int e = find_entry(descs, count, blockIdx.x);
  const ApplyDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  constexpr int CPR = kApplyCols / 8, RPP = 256 / CPR;
  const int64_t row0 = int64_t(lt / d.tiles_n) * kApplyRows, col0 = int64_t(lt % d.tiles_n) * kApplyCols;
  const int t = threadIdx.x;
  const int c8 = (t % CPR) * 8, rr = t / CPR;
  const float osc = d.use_scale ? d.scale[0] : 1.0f;
  const int64_t m = d.m, n = d.n;
  const bool vec = (n % 8 == 0);
#pragma unroll
  for (int q = 0; q < kApplyRows / RPP; ++q) {
    const int64_t i = row0 + rr + RPP * q;
    const int64_t j0 = col0 + c8;
    if (i >= m || j0 >= n) continue;
    V8 o;
    load8<NSDT, true>(d.o, blk_index(i, j0, d.ld_o), o);  // j0 < n: the padded O row holds these 8 columns
#pragma unroll
    for (int k = 0; k < 8; ++k) o.v[k] *= osc;
    const int64_t idx = i * n + j0;
    if (vec && j0 + 7 < n) {
      if (d.mode == 0) {
        V8 p;
        if (d.param_dtype == kDtBF16) load8<kDtBF16, true>(d.param, idx, p); else load8<kDtF32, true>(d.param, idx, p);
#pragma unroll
        for (int k = 0; k < 8; ++k) p.v[k] = p.v[k] * d.decay - d.step * o.v[k];
        if (d.param_dtype == kDtBF16) store8<kDtBF16, true>(d.param, idx, p); else store8<kDtF32, true>(d.param, idx, p);
        if (d.update_out) store8<kDtF32, true>(d.update_out, idx, o);
      } else {
        if (d.param_dtype == kDtBF16) store8<kDtBF16, true>(d.param, idx, o); else store8<kDtF32, true>(d.param, idx, o);
      }
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (j0 + k >= n) break;
        if (d.mode == 0) {
          const float p = load_as_f32(d.param, idx + k, d.param_dtype);
          store_from_f32(d.param, idx + k, p * d.decay - d.step * o.v[k], d.param_dtype);
          if (d.update_out) d.update_out[idx + k] = o.v[k];
        } else {
          store_from_f32(d.param, idx + k, o.v[k], d.param_dtype);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// AdamW: grouped over up to kAdamWMaxPerLaunch tensors passed by value; each workgroup owns
// kAdamWBlockElems consecutive elements of one tensor, in 8-element (16-B bf16) vectors.
__device__ __forceinline__ void adamw_elem(float& p, float g, float& m, float& v, const AdamWBatch& b) {
  p = p * b.decay;
  m = m + b.omb1 * (g - m);
  v = b.beta2 * v + b.omb2 * g * g;
  const float denom = sqrtf(v) * b.inv_sqrt_bc2 + b.eps;
  p = p - b.step_size * (m / denom);
}

constexpr bool kAdamWNtLoad = false;   // non-temporal loads / stores of the AdamW streams
constexpr bool kAdamWNtStore = false;

__global__ __launch_bounds__(256) void adamw_kernel(const AdamWBatch batch) {
  int e = 0;
  for (int k = 1; k < batch.count; ++k)
    if (batch.d[k].block_begin <= int(blockIdx.x)) e = k;
  const AdamWDesc& d = batch.d[e];
  const int64_t base = int64_t(blockIdx.x - d.block_begin) * kAdamWBlockElems;
  constexpr int NQ = kAdamWBlockElems / 2048;
  // thread t owns elements base + (q * 256 + t) * 8 .. +7, q = 0 .. NQ - 1
  if (base + kAdamWBlockElems <= d.numel) {
    // whole block inside the tensor: every load of the block is issued before the first store
    auto run = [&](auto pdt, auto gdt) {
      constexpr int PDT = decltype(pdt)::value, GDT = decltype(gdt)::value;
      V8 p[NQ], g[NQ], m[NQ], v[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int64_t i0 = base + (int64_t(q) * 256 + threadIdx.x) * 8;
        load8<PDT, kAdamWNtLoad>(d.param, i0, p[q]);
        load8<GDT, kAdamWNtLoad>(d.grad, i0, g[q]);
        load8<kDtF32, kAdamWNtLoad>(d.exp_avg, i0, m[q]);
        load8<kDtF32, kAdamWNtLoad>(d.exp_avg_sq, i0, v[q]);
      }
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int64_t i0 = base + (int64_t(q) * 256 + threadIdx.x) * 8;
#pragma unroll
        for (int k = 0; k < 8; ++k) adamw_elem(p[q].v[k], g[q].v[k], m[q].v[k], v[q].v[k], batch);
        store8<PDT, kAdamWNtStore>(d.param, i0, p[q]);
        store8<kDtF32, kAdamWNtStore>(d.exp_avg, i0, m[q]);
        store8<kDtF32, kAdamWNtStore>(d.exp_avg_sq, i0, v[q]);
      }
    };
    using BF = std::integral_constant<int, kDtBF16>;
    using F32 = std::integral_constant<int, kDtF32>;
    if (d.param_dtype == kDtBF16) {
      if (d.grad_dtype == kDtBF16) run(BF{}, BF{}); else run(BF{}, F32{});
    } else {
      if (d.grad_dtype == kDtBF16) run(F32{}, BF{}); else run(F32{}, F32{});
    }
    return;
  }
  for (int q = 0; q < NQ; ++q) {
    const int64_t i0 = base + (int64_t(q) * 256 + threadIdx.x) * 8;
    if (i0 >= d.numel) break;
    if (i0 + 7 < d.numel) {
      V8 p, g, m, v;
      if (d.param_dtype == kDtBF16) load8<kDtBF16>(d.param, i0, p); else load8<kDtF32>(d.param, i0, p);
      if (d.grad_dtype == kDtBF16) load8<kDtBF16>(d.grad, i0, g); else load8<kDtF32>(d.grad, i0, g);
      load8<kDtF32>(d.exp_avg, i0, m);
      load8<kDtF32>(d.exp_avg_sq, i0, v);
#pragma unroll
      for (int k = 0; k < 8; ++k) adamw_elem(p.v[k], g.v[k], m.v[k], v.v[k], batch);
      if (d.param_dtype == kDtBF16) store8<kDtBF16>(d.param, i0, p); else store8<kDtF32>(d.param, i0, p);
      store8<kDtF32>(d.exp_avg, i0, m);
      store8<kDtF32>(d.exp_avg_sq, i0, v);
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
                       int reduce, float beta, float one_minus_beta, int nesterov, hipStream_t st) {
  if (total_tiles <= 0) return hipSuccess;
  if (reduce) {
    if (ns_dtype == kDtBF16)
      hipLaunchKernelGGL((prep_kernel<kDtBF16, true>), dim3(total_tiles), dim3(256), 0, st, d_descs,
                         count, beta, one_minus_beta, nesterov);
    else
      hipLaunchKernelGGL((prep_kernel<kDtF32, true>), dim3(total_tiles), dim3(256), 0, st, d_descs,
                         count, beta, one_minus_beta, nesterov);
    return hipGetLastError();
  }
  if (ns_dtype == kDtBF16)
    hipLaunchKernelGGL((prep_kernel<kDtBF16, false>), dim3(total_tiles), dim3(256), 0, st, d_descs,
                       count, beta, one_minus_beta, nesterov);
  else
    hipLaunchKernelGGL((prep_kernel<kDtF32, false>), dim3(total_tiles), dim3(256), 0, st, d_descs,
                       count, beta, one_minus_beta, nesterov);
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
