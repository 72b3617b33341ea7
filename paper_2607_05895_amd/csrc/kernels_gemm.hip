// Newton-Schulz products on gfx950.
//
// Every product of the quintic step is computed as one grouped "NT" GEMM
//     C = alpha * P Q^T + beta * E        (P: M x K, Q: N x K, both row-major, K-contiguous)
// over all matrices of the owner in one launch (one problem per matrix, tiles of all problems
// enumerated heaviest-K first). Symmetric products (A = X X^T and A A) compute only the tiles on
// and above the diagonal and store each off-diagonal tile twice (as is and transposed).
//
// bf16 path: 256 x 256 output tile per workgroup of 4 waves (2 x 2), 128 x 128 per wave as 4 x 4
// v_mfma_f32_32x32x16_bf16 blocks with fp32 accumulation; K step 64 staged through LDS (two
// stages of 64 KiB) with an XOR swizzle of 16-byte chunks so that fragment reads are free of bank
// conflicts. The next K step's global loads are in flight while the current one is multiplied.
// fp32 path: 64 x 64 tiles on the vector ALUs (a correctness path for fp32 NS).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfsdp_internal.h"

namespace mfsdp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  auto cvt = [](float f) -> uint32_t {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
  };
  return cvt(lo) | (cvt(hi) << 16);
}

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

template <typename D>
__device__ __forceinline__ int find_entry(const D* descs, int count, int key) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (descs[mid].tile_begin <= key) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Map a problem-local tile index to (bi, bj): row-major over the full grid, or over the upper
// triangle (bi <= bj) for symmetric products.
__device__ __forceinline__ void tile_coords(const GemmDesc& d, int lt, int& bi, int& bj) {
  if (d.sym) {
    const int T = d.tiles_m;
    int r = 0, rem = lt;
    while (rem >= T - r) { rem -= T - r; ++r; }
    bi = r;
    bj = r + rem;
  } else {
    bi = lt / d.tiles_n;
    bj = lt % d.tiles_n;
  }
}

__device__ __forceinline__ float scale_pow(const float* s, int pw) {
  if (!s || pw == 0) return 1.0f;
  const float v = *s;
  return pw == 1 ? v : v * v;
}

// ---------------------------------------------------------------------------------------------
// bf16 MFMA kernel
constexpr int BT = 256;             // output tile (both sides)
constexpr int BKE = 64;             // K elements per stage
constexpr int ROWB = BKE * 2;       // bytes per staged row (128)
constexpr int STAGE_BYTES = 2 * BT * ROWB;  // P rows then Q rows: 64 KiB

__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(const GemmDesc* __restrict__ descs,
                                                           int count, int parity, int first,
                                                           int last) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE_BYTES];

  const int e = find_entry(descs, count, blockIdx.x);
  const GemmDesc& dd = descs[e];
  const int lt = blockIdx.x - dd.tile_begin;
  int bi, bj;
  tile_coords(dd, lt, bi, bj);
  const uint16_t* __restrict__ P = static_cast<const uint16_t*>(dd.P[parity]);
  const uint16_t* __restrict__ Q = static_cast<const uint16_t*>(dd.Q[parity]);
  const int64_t ldp = dd.ldp, ldq = dd.ldq;
  const int K = dd.K;

  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int wm = w >> 1, wn = w & 1;

  // Loader: thread t covers staged rows c * 32 + t / 8 (c = 0..15; rows 0..255 are P, 256..511
  // are Q) and 16-byte slot t % 8 of each row; the slot holds global chunk slot ^ (row % 8).
  const int lrow = t >> 3, lslot = t & 7;
  const int lchunk = lslot ^ (lrow & 7);
  // rows c*32 + lrow: c < 8 from P, c >= 8 from Q; consecutive c are 32 rows apart
  const uint16_t* psrc = P + (int64_t(bi) * BT + lrow) * ldp + lchunk * 8;
  const uint16_t* qsrc = Q + (int64_t(bj) * BT + lrow) * ldq + lchunk * 8;
  const int64_t pstep = 32 * ldp, qstep = 32 * ldq;
  const int lds_w_off = lrow * ROWB + lslot * 16;  // + c * 32 * ROWB

  f32x16_t acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

  const int nk = K / BKE;
  // fragment read offsets: row (base + l%32), chunk q = 2*kk + l/32, slot q ^ (l % 8)
  const int frow = lane & 31, fhalf = lane >> 5;
  const int pbase = (wm * 128 + frow) * ROWB;
  const int qbase = (BT + wn * 128 + frow) * ROWB;

  uint4 s0, s1, s2, s3, s4, s5, s6, s7, s8, s9, s10, s11, s12, s13, s14, s15;
#define MFSDP_GLOAD(koff)                                                                \
  do {                                                                                   \
    const uint16_t* pp = psrc + (koff);                                                  \
    const uint16_t* qq = qsrc + (koff);                                                  \
    s0 = *reinterpret_cast<const uint4*>(pp);                                            \
    s1 = *reinterpret_cast<const uint4*>(pp + pstep);                                    \
    s2 = *reinterpret_cast<const uint4*>(pp + 2 * pstep);                                \
    s3 = *reinterpret_cast<const uint4*>(pp + 3 * pstep);                                \
    s4 = *reinterpret_cast<const uint4*>(pp + 4 * pstep);                                \
    s5 = *reinterpret_cast<const uint4*>(pp + 5 * pstep);                                \
    s6 = *reinterpret_cast<const uint4*>(pp + 6 * pstep);                                \
    s7 = *reinterpret_cast<const uint4*>(pp + 7 * pstep);                                \
    s8 = *reinterpret_cast<const uint4*>(qq);                                            \
    s9 = *reinterpret_cast<const uint4*>(qq + qstep);                                    \
    s10 = *reinterpret_cast<const uint4*>(qq + 2 * qstep);                               \
    s11 = *reinterpret_cast<const uint4*>(qq + 3 * qstep);                               \
    s12 = *reinterpret_cast<const uint4*>(qq + 4 * qstep);                               \
    s13 = *reinterpret_cast<const uint4*>(qq + 5 * qstep);                               \
    s14 = *reinterpret_cast<const uint4*>(qq + 6 * qstep);                               \
    s15 = *reinterpret_cast<const uint4*>(qq + 7 * qstep);                               \
  } while (0)
#define MFSDP_LSTORE(buf)                                                                \
  do {                                                                                   \
    uint8_t* b_ = (buf) + lds_w_off;                                                     \
    *reinterpret_cast<uint4*>(b_ + 0 * 32 * ROWB) = s0;                                  \
    *reinterpret_cast<uint4*>(b_ + 1 * 32 * ROWB) = s1;                                  \
    *reinterpret_cast<uint4*>(b_ + 2 * 32 * ROWB) = s2;                                  \
    *reinterpret_cast<uint4*>(b_ + 3 * 32 * ROWB) = s3;                                  \
    *reinterpret_cast<uint4*>(b_ + 4 * 32 * ROWB) = s4;                                  \
    *reinterpret_cast<uint4*>(b_ + 5 * 32 * ROWB) = s5;                                  \
    *reinterpret_cast<uint4*>(b_ + 6 * 32 * ROWB) = s6;                                  \
    *reinterpret_cast<uint4*>(b_ + 7 * 32 * ROWB) = s7;                                  \
    *reinterpret_cast<uint4*>(b_ + 8 * 32 * ROWB) = s8;                                  \
    *reinterpret_cast<uint4*>(b_ + 9 * 32 * ROWB) = s9;                                  \
    *reinterpret_cast<uint4*>(b_ + 10 * 32 * ROWB) = s10;                                \
    *reinterpret_cast<uint4*>(b_ + 11 * 32 * ROWB) = s11;                                \
    *reinterpret_cast<uint4*>(b_ + 12 * 32 * ROWB) = s12;                                \
    *reinterpret_cast<uint4*>(b_ + 13 * 32 * ROWB) = s13;                                \
    *reinterpret_cast<uint4*>(b_ + 14 * 32 * ROWB) = s14;                                \
    *reinterpret_cast<uint4*>(b_ + 15 * 32 * ROWB) = s15;                                \
  } while (0)

  // Fragments of K-slice kk + 1 are read while the 16 MFMAs of slice kk run.
  auto compute = [&](const uint8_t* sb) {
    bf16x8_t pf[2][4], qf[2][4];
    auto read_frags = [&](int kk, int b) {
      const int slot = ((2 * kk + fhalf) ^ (lane & 7)) * 16;
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        pf[b][mi] = *reinterpret_cast<const bf16x8_t*>(sb + pbase + mi * 32 * ROWB + slot);
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
        qf[b][ni] = *reinterpret_cast<const bf16x8_t*>(sb + qbase + ni * 32 * ROWB + slot);
    };
    read_frags(0, 0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (kk < 3) read_frags(kk + 1, (kk + 1) & 1);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[kk & 1][ni], pf[kk & 1][mi],
                                                                acc[mi][ni], 0, 0, 0);
    }
  };

  MFSDP_GLOAD(0);
  MFSDP_LSTORE(smem);
  __syncthreads();
  for (int kt = 0; kt + 1 < nk; ++kt) {
    const int cur = kt & 1;
    MFSDP_GLOAD(int64_t(kt + 1) * BKE);
    compute(smem + cur * STAGE_BYTES);
    MFSDP_LSTORE(smem + (cur ^ 1) * STAGE_BYTES);
    __syncthreads();
  }
  compute(smem + ((nk - 1) & 1) * STAGE_BYTES);
#undef MFSDP_GLOAD
#undef MFSDP_LSTORE

  // Epilogue. acc[mi][ni] holds D[j][i] = C[i][j] with i = i0 + lane % 32 and
  // j = j0 + 8 g + 4 (lane / 32) + t for element v = 4 g + t.
  const float alpha = dd.alpha * (first ? scale_pow(dd.scale, dd.alpha_scale_pow) : 1.0f);
  const float beta = dd.beta * (first ? scale_pow(dd.scale, dd.beta_scale_pow) : 1.0f);
  const uint16_t* E = static_cast<const uint16_t*>(dd.E[parity]);
  uint16_t* C = static_cast<uint16_t*>(dd.C[parity]);
  uint16_t* CT = static_cast<uint16_t*>(dd.CT[parity]);
  if (last) {
    if (!dd.last_c) C = nullptr;
    if (!dd.last_ct) CT = nullptr;
  }
  const bool mirror = dd.sym && bi != bj && C;
  const int64_t lde = dd.lde, ldc = dd.ldc, ldct = dd.ldct;
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int64_t i = int64_t(bi) * BT + wm * 128 + mi * 32 + frow;
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int64_t j = int64_t(bj) * BT + wn * 128 + ni * 32 + g * 8 + fhalf * 4;
        float v0 = alpha * acc[mi][ni][4 * g + 0];
        float v1 = alpha * acc[mi][ni][4 * g + 1];
        float v2 = alpha * acc[mi][ni][4 * g + 2];
        float v3 = alpha * acc[mi][ni][4 * g + 3];
        if (E) {
          const uint2 ev = *reinterpret_cast<const uint2*>(E + i * lde + j);
          v0 += beta * __uint_as_float(ev.x << 16);
          v1 += beta * __uint_as_float(ev.x & 0xffff0000u);
          v2 += beta * __uint_as_float(ev.y << 16);
          v3 += beta * __uint_as_float(ev.y & 0xffff0000u);
        }
        const uint32_t w01 = pack_bf16x2(v0, v1), w23 = pack_bf16x2(v2, v3);
        if (C) {
          *reinterpret_cast<uint2*>(C + i * ldc + j) = make_uint2(w01, w23);
          if (mirror) {
            C[(j + 0) * ldc + i] = uint16_t(w01);
            C[(j + 1) * ldc + i] = uint16_t(w01 >> 16);
            C[(j + 2) * ldc + i] = uint16_t(w23);
            C[(j + 3) * ldc + i] = uint16_t(w23 >> 16);
          }
        }
        if (CT) {
          CT[(j + 0) * ldct + i] = uint16_t(w01);
          CT[(j + 1) * ldct + i] = uint16_t(w01 >> 16);
          CT[(j + 2) * ldct + i] = uint16_t(w23);
          CT[(j + 3) * ldct + i] = uint16_t(w23 >> 16);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// fp32 kernel: 64 x 64 tile, 256 threads of 4 x 4 outputs, K step 16 through LDS.
__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmDesc* __restrict__ descs, int count,
                                                       int parity, int first, int last) {
  __shared__ float Ps[16][68];
  __shared__ float Qs[16][68];
  const int e = find_entry(descs, count, blockIdx.x);
  const GemmDesc& dd = descs[e];
  const int lt = blockIdx.x - dd.tile_begin;
  int bi, bj;
  tile_coords(dd, lt, bi, bj);
  const float* __restrict__ P = static_cast<const float*>(dd.P[parity]);
  const float* __restrict__ Q = static_cast<const float*>(dd.Q[parity]);
  const int t = threadIdx.x;
  const int tx = t & 15, ty = t >> 4;
  const int lr = t >> 2, lk = (t & 3) * 4;
  const float* psrc = P + (int64_t(bi) * 64 + lr) * dd.ldp + lk;
  const float* qsrc = Q + (int64_t(bj) * 64 + lr) * dd.ldq + lk;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < dd.K; k0 += 16) {
    const float4 pv = *reinterpret_cast<const float4*>(psrc + k0);
    const float4 qv = *reinterpret_cast<const float4*>(qsrc + k0);
    Ps[lk + 0][lr] = pv.x; Ps[lk + 1][lr] = pv.y; Ps[lk + 2][lr] = pv.z; Ps[lk + 3][lr] = pv.w;
    Qs[lk + 0][lr] = qv.x; Qs[lk + 1][lr] = qv.y; Qs[lk + 2][lr] = qv.z; Qs[lk + 3][lr] = qv.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float4 a = *reinterpret_cast<const float4*>(&Ps[k][ty * 4]);
      const float4 b = *reinterpret_cast<const float4*>(&Qs[k][tx * 4]);
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(av[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
  const float alpha = dd.alpha * (first ? scale_pow(dd.scale, dd.alpha_scale_pow) : 1.0f);
  const float beta = dd.beta * (first ? scale_pow(dd.scale, dd.beta_scale_pow) : 1.0f);
  const float* E = static_cast<const float*>(dd.E[parity]);
  float* C = static_cast<float*>(dd.C[parity]);
  float* CT = static_cast<float*>(dd.CT[parity]);
  if (last) {
    if (!dd.last_c) C = nullptr;
    if (!dd.last_ct) CT = nullptr;
  }
  const bool mirror = dd.sym && bi != bj && C;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = int64_t(bi) * 64 + ty * 4 + r;
    const int64_t j = int64_t(bj) * 64 + tx * 4;
    float v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = alpha * acc[r][c];
    if (E) {
      const float4 ev = *reinterpret_cast<const float4*>(E + i * dd.lde + j);
      v[0] += beta * ev.x; v[1] += beta * ev.y; v[2] += beta * ev.z; v[3] += beta * ev.w;
    }
    if (C) {
      *reinterpret_cast<float4*>(C + i * dd.ldc + j) = make_float4(v[0], v[1], v[2], v[3]);
      if (mirror)
#pragma unroll
        for (int c = 0; c < 4; ++c) C[(j + c) * dd.ldc + i] = v[c];
    }
    if (CT)
#pragma unroll
      for (int c = 0; c < 4; ++c) CT[(j + c) * dd.ldct + i] = v[c];
  }
}

}  // namespace

hipError_t launch_gemm(const GemmDesc* d_descs, int count, int total_tiles, int ns_dtype,
                       int parity, int first_step, int last_step, hipStream_t st) {
  if (total_tiles <= 0) return hipSuccess;
  if (ns_dtype == kDtBF16)
    hipLaunchKernelGGL(gemm_bf16_kernel, dim3(total_tiles), dim3(256), 0, st, d_descs, count,
                       parity, first_step, last_step);
  else
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(total_tiles), dim3(256), 0, st, d_descs, count,
                       parity, first_step, last_step);
  return hipGetLastError();
}

}  // namespace mfsdp
