// HIP kernels of the Shampoo owner step (fp32): the NT GEMM on fp32 MFMA that every product of the
// step reduces to (statistics G G^T and G^T G, the coupled Newton iteration for the inverse root,
// P_L G P_R), and the small boundary, reduction and elementwise kernels around it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "mfsdp_internal.h"
#include "shampoo_internal.h"

namespace mfsdp {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
// global-address-space views (flat accesses would also count against the LDS wait counter)
typedef __attribute__((address_space(1))) float g_f32;
typedef __attribute__((address_space(1))) const float g_cf32;
typedef __attribute__((address_space(1))) const f32x4 g_cf32x4;

// The descriptor serving block b (descriptors sorted by tile_begin, the first one at 0).
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

__device__ __forceinline__ float ld_any(const void* p, int64_t i, int dt) {
  if (dt == kDtBF16) return __uint_as_float(uint32_t(static_cast<const uint16_t*>(p)[i]) << 16);
  return static_cast<const float*>(p)[i];
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Exact three-way split of four fp32 values into bf16 parts, x = hi + mid + lo (4 bf16 each, packed
// in two dwords): hi is x rounded to bf16 (nearest even), mid the rounded remainder, lo the rounded
// second remainder. Each remainder is exact in fp32 (it is x's lower bits), so only lo rounds, at
// about 2^-25 |x|.
__device__ __forceinline__ void split3x4(const f32x4& x, u32x2& hi, u32x2& mid, u32x2& lo) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const uint32_t h = pack_bf16x2(x[2 * j], x[2 * j + 1]);
    hi[j] = h;
    const float a = x[2 * j] - __uint_as_float(h << 16);
    const float b = x[2 * j + 1] - __uint_as_float(h & 0xffff0000u);
    const uint32_t m = pack_bf16x2(a, b);
    mid[j] = m;
    lo[j] = pack_bf16x2(a - __uint_as_float(m << 16), b - __uint_as_float(m & 0xffff0000u));
  }
}

// 16-byte slot of (row r, k-chunk c) in a split operand plane (rows of 16 bf16 = two 16-byte
// chunks): c ^ ((r >> 3) & 1), so that 16 consecutive rows at one chunk (a quarter wave's fragment
// reads) fall in 16 distinct 16-byte bank groups, and a wave's 8-byte stores (4 lanes per row) in 32.
__device__ __forceinline__ int split_slot(int r, int c) { return r * 2 + (c ^ ((r >> 3) & 1)); }

constexpr int kShPlane = kShTile * 32;  // bytes of one split plane (128 x 16 bf16)
constexpr int kShStage = 6 * kShPlane;  // both operands of one K step, three planes each

// The products of one 128 x 128 output tile, P rows from bi, Q rows from bj, into acc. An fp32
// operand is split into three bf16 parts (hi + mid + lo); an operand stored as bf16 (ABF, BBF: a
// bf16 gradient) is its own single part, as if its mid and lo parts were zero: the products with
// them are dropped, which leaves the accumulated sums unchanged. It is loaded as it is, 8 bytes per
// 4 elements, and stored into its plane without a split.
// 4 waves in a 2 x 2 arrangement, each 64 x 64 as 2 x 2 blocks of 32 x 32 outputs. The products
// run on the bf16 MFMA (v_mfma_f32_32x32x16_bf16, fp32 accumulation) at fp32 accuracy: when a
// K step of 16 is staged into LDS every element is split once into hi + mid + lo bf16 parts (three
// planes per operand); a lane's fragment is 8 consecutive k of one row from each plane, and the
// six partial products above 2^-24 relative are accumulated (lo.hi, hi.lo, mid.mid, mid.hi, hi.mid,
// hi.hi; the dropped mid.lo, lo.mid, lo.lo are below 2^-32). Six bf16 MFMAs per 16 k take 192
// cycles against 512 for the fp32 MFMA.
// A stage holds KS K steps (KS (PA + PB) planes, at most six: 24 KiB); the LDS is double
// buffered, and two register sets hold the global loads of the next two stages, so that the loads
// of stage k + 2 are issued while stage k multiplies and stage k + 1's loads (issued a stage
// earlier) are split into LDS. Few products per step (one-part operands) take several steps per
// stage, so that a barrier and the load latency are spread over more MFMAs.
template <bool ABF, bool BBF>
__device__ __forceinline__ void sh_tile_products(const ShGemmDesc& d, int bi, int bj, uint8_t* lds_raw,
                                                 f32x16 (&acc)[2][2]) {
  constexpr int PA = ABF ? 1 : 3, PB = BBF ? 1 : 3;  // parts per operand
  constexpr int KS = ABF && BBF ? 2 : 1;             // K steps per stage
  static_assert(KS * (PA + PB) <= 6, "a stage holds at most six planes");
  typedef __attribute__((address_space(1))) const uint8_t g_cu8;
  typedef __attribute__((address_space(1))) const u32x2 g_cu32x2;
  constexpr int ea = ABF ? 2 : 4, eb = BBF ? 2 : 4;  // bytes per element
  using TA = typename std::conditional<ABF, u32x2, f32x4>::type;
  using TB = typename std::conditional<BBF, u32x2, f32x4>::type;
  // tile rows of both operands (uniform) and this thread's byte offsets into them (32-bit: a tile
  // spans at most 128 rows with a row stride of at most 2 x 65536 elements, under 2^27 bytes)
  g_cu8* P = (g_cu8*)(d.P) + int64_t(bi) * kShTile * d.ldp * ea;
  g_cu8* Q = (g_cu8*)(d.Q) + int64_t(bj) * kShTile * d.ldq * eb;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int fr = lane & 31, fh = lane >> 5;
  // staging: thread t loads k 4 (t & 3) .. + 3 of each step of rows t / 4 and t / 4 + 64 of both
  // operands
  const int lrow = t >> 2, lch = t & 3;
  uint32_t po[2], qo[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    po[j] = uint32_t((lrow + 64 * j) * d.ldp + lch * 4) * uint32_t(ea);
    qo[j] = uint32_t((lrow + 64 * j) * d.ldq + lch * 4) * uint32_t(eb);
  }
  TA ra0[KS][2], ra1[KS][2];
  TB rb0[KS][2], rb1[KS][2];
  auto gload = [&](TA (&ra)[KS][2], TB (&rb)[KS][2], int k0) {
#pragma unroll
    for (int u = 0; u < KS; ++u)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if constexpr (ABF) ra[u][j] = *(g_cu32x2*)(P + (k0 + 16 * u) * ea + po[j]);
        else ra[u][j] = *(const g_cf32x4*)(P + (k0 + 16 * u) * ea + po[j]);
        if constexpr (BBF) rb[u][j] = *(g_cu32x2*)(Q + (k0 + 16 * u) * eb + qo[j]);
        else rb[u][j] = *(const g_cf32x4*)(Q + (k0 + 16 * u) * eb + qo[j]);
      }
  };
  // plane (step u, operand o, part p) of a stage is u (PA + PB) + o PA + p; the 8-byte piece of
  // row r holding k 4 lch .. + 3
  auto plane = [](int u, int o, int p) { return u * (PA + PB) + o * PA + p; };
  auto lstore = [&](int s, const TA (&ra)[KS][2], const TB (&rb)[KS][2]) {
#pragma unroll
    for (int u = 0; u < KS; ++u)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int r = lrow + 64 * j;
        const int off = split_slot(r, lch >> 1) * 16 + (lch & 1) * 8;
        uint8_t* base = lds_raw + s * kShStage + off;
        u32x2 h, m, l;
        if constexpr (ABF) {
          *reinterpret_cast<u32x2*>(base + plane(u, 0, 0) * kShPlane) = ra[u][j];
        } else {
          split3x4(ra[u][j], h, m, l);
          *reinterpret_cast<u32x2*>(base + plane(u, 0, 0) * kShPlane) = h;
          *reinterpret_cast<u32x2*>(base + plane(u, 0, 1) * kShPlane) = m;
          *reinterpret_cast<u32x2*>(base + plane(u, 0, 2) * kShPlane) = l;
        }
        if constexpr (BBF) {
          *reinterpret_cast<u32x2*>(base + plane(u, 1, 0) * kShPlane) = rb[u][j];
        } else {
          split3x4(rb[u][j], h, m, l);
          *reinterpret_cast<u32x2*>(base + plane(u, 1, 0) * kShPlane) = h;
          *reinterpret_cast<u32x2*>(base + plane(u, 1, 1) * kShPlane) = m;
          *reinterpret_cast<u32x2*>(base + plane(u, 1, 2) * kShPlane) = l;
        }
      }
  };
  auto frag = [&](int s, int pl, int r) {
    return *reinterpret_cast<const bf16x8_t*>(lds_raw + s * kShStage + pl * kShPlane + split_slot(r, fh) * 16);
  };
  // parts 0, 1, 2 = hi, mid, lo; the six products (lo.hi, hi.lo, mid.mid, mid.hi, hi.mid, hi.hi)
  // term by term over the four blocks, so that consecutive MFMAs use different accumulators
  auto mfma_stage = [&](int s) {
#pragma unroll
    for (int u = 0; u < KS; ++u) {
      bf16x8_t af[2][PA], bf[2][PB];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int pt = 0; pt < PA; ++pt) af[i][pt] = frag(s, plane(u, 0, pt), wr * 64 + i * 32 + fr);
#pragma unroll
        for (int pt = 0; pt < PB; ++pt) bf[i][pt] = frag(s, plane(u, 1, pt), wc * 64 + i * 32 + fr);
      }
      constexpr int kTerm[6][2] = {{2, 0}, {0, 2}, {1, 1}, {1, 0}, {0, 1}, {0, 0}};
#pragma unroll
      for (int tm = 0; tm < 6; ++tm) {
        if (kTerm[tm][0] >= PA || kTerm[tm][1] >= PB) continue;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i][kTerm[tm][0]], bf[j][kTerm[tm][1]],
                                                                acc[i][j], 0, 0, 0);
      }
    }
  };
  constexpr int kStep = 16 * KS;  // k per stage
  constexpr int kTerms = PA == 3 && PB == 3 ? 6 : PA == 3 || PB == 3 ? 3 : 1;
  constexpr int kMfma = KS * 4 * kTerms;  // MFMAs per stage and wave
  constexpr int kSplitValu = KS * 2 * ((ABF ? 0 : 22) + (BBF ? 0 : 22));  // split VALU per stage, about
  // one stage's products on LDS buffer mb while the next stage's loads (set) are split into buffer
  // sb: with split operands the split's vector instructions and LDS stores are interleaved with the
  // MFMAs (they are independent), so that a wave's MFMA pipe and vector ALU work at the same time
  // (one-part products have little to interleave and run faster in program order)
  auto stage = [&](int mb, int sb, const TA (&ra)[KS][2], const TB (&rb)[KS][2]) {
    mfma_stage(mb);
    lstore(sb, ra, rb);
    if constexpr (kTerms > 1) {
      constexpr int kV = (kSplitValu + kMfma - 1) / kMfma;
#pragma unroll
      for (int i = 0; i < kMfma; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // 1 MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, kV, 0);  // vector ALU
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);   // LDS store
      }
    }
  };
  // K is a multiple of 128, so nk is even and at least 4: even stages live in LDS buffer 0 and
  // register set 0, odd ones in buffer 1 and set 1, and the loads run two stages ahead
  const int nk = d.K / kStep;
  gload(ra0, rb0, 0);
  gload(ra1, rb1, kStep);
  lstore(0, ra0, rb0);
  __syncthreads();
  int kt = 0;
  for (; kt + 2 < nk; kt += 2) {
    gload(ra0, rb0, (kt + 2) * kStep);
    stage(0, 1, ra1, rb1);
    __syncthreads();
    gload(ra1, rb1, (kt + 3) * kStep);
    stage(1, 0, ra0, rb0);
    __syncthreads();
  }
  stage(0, 1, ra1, rb1);
  __syncthreads();
  mfma_stage(1);
  __syncthreads();
}

// C = alpha P Q^T + beta E + diag I on one 128 x 128 output tile per workgroup (products as in
// sh_tile_products, with the descriptor's operand types: both bf16, Q bf16, or both fp32). 48 KiB of LDS lets three workgroups share a CU.
// Symmetric problems compute the upper tiles only and store each tile transposed as well, through
// LDS, with coalesced row stores.
__global__ __launch_bounds__(256, 3) void sh_gemm_kernel(const ShGemmDesc* __restrict__ descs, int count) {
  __shared__ __attribute__((aligned(16))) uint8_t lds_raw[2 * kShStage];
  const int e = find_desc(descs, count, blockIdx.x);
  const ShGemmDesc& d = descs[e];
  int lt = blockIdx.x - d.tile_begin;
  if (d.clear && lt == 0 && threadIdx.x == 0) *d.clear = 0.0f;
  int bi, bj;
  if (d.sym) {
    bi = 0;
    int rowlen = d.tiles_n;
    while (lt >= rowlen) {
      lt -= rowlen;
      ++bi;
      --rowlen;
    }
    bj = bi + lt;
  } else {
    bi = lt / d.tiles_n;
    bj = lt - bi * d.tiles_n;
  }
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int fr = lane & 31, fh = lane >> 5;
  if (d.conv_in && *d.conv_in < kShConvTol) {  // converged side: the iterate no longer changes
    if (d.copy_on_skip) {
      const g_cf32* src = (const g_cf32*)(d.E);
      g_f32* dst = (g_f32*)(d.C);
#pragma unroll 4
      for (int it = 0; it < 64; ++it) {
        const int r = (t >> 7) + 2 * it, c = t & 127;
        dst[(int64_t(bi) * kShTile + r) * d.ldc + int64_t(bj) * kShTile + c] =
            src[(int64_t(bi) * kShTile + r) * d.lde + int64_t(bj) * kShTile + c];
        if (bi != bj)
          dst[(int64_t(bj) * kShTile + r) * d.ldc + int64_t(bi) * kShTile + c] =
              src[(int64_t(bj) * kShTile + r) * d.lde + int64_t(bi) * kShTile + c];
      }
    }
    return;
  }
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  if (d.q_bf16 && d.p_bf16)
    sh_tile_products<true, true>(d, bi, bj, lds_raw, acc);
  else if (d.q_bf16)
    sh_tile_products<false, true>(d, bi, bj, lds_raw, acc);
  else
    sh_tile_products<false, false>(d, bi, bj, lds_raw, acc);

  // Epilogue, in two passes over the tile's row halves (the waves with wr = h hold rows
  // 64 h .. 64 h + 63). Accumulator element v of block (i, j) is row 32 i + 8 (v / 4) + 4 (lane / 32)
  // + v % 4 of the half, column 64 wc + 32 j + lane % 32. E's half (which may alias C) is first
  // copied into LDS by direct global->LDS loads (64 x 128 fp32 = 32 KiB, rows of 512 B), so that no
  // store of C waits for an E load behind it; every element of E used is read before the element is
  // written, by the same thread. The final values stay in acc for the transposed stores.
  // Symmetric problems are stored exactly symmetric: an upper tile is also stored transposed,
  // through a 64 x 128 LDS tile per half (element (rl, c) at rl * 128 + (c ^ rl)), and a diagonal
  // tile keeps its upper triangle and mirrors it into the lower one (in floating point the two
  // triangles of a product of two different symmetric matrices differ; kept, that antisymmetric
  // part is amplified by the NT form of the iteration). The lower triangle of a diagonal tile's E
  // may be overwritten by the first half's mirror before the second half is copied; it is not used.
  typedef __attribute__((address_space(3))) uint8_t lds_u8;
  g_f32* C = (g_f32*)(d.C);
  const g_cf32* E = (const g_cf32*)(d.E);
  const bool diag_tile = d.sym && bi == bj;
  const int64_t r0 = int64_t(bi) * kShTile, c0 = int64_t(bj) * kShTile;
  float* tl = reinterpret_cast<float*>(lds_raw);
  float res = 0.0f;  // max |C - I| over this thread's elements of the real block
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h == 1 && (E || d.sym)) __syncthreads();  // the first half's LDS reads are done
    if (E) {
      // wave w copies rows 16 w .. 16 w + 15 of the half, two rows (1 KiB) per instruction (a
      // uniform row base and 32-bit lane offsets)
      typedef __attribute__((address_space(1))) const uint8_t g_cu8e;
      g_cu8e* eb = (g_cu8e*)(E + (r0 + 64 * h + 16 * w) * d.lde + c0);
      const uint32_t eo = uint32_t(((lane >> 5) * d.lde + 4 * (lane & 31)) * 4);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_global_load_lds((const void*)(eb + 2 * i * d.lde * 4 + eo),
                                         (lds_u8*)(lds_raw + (16 * w + 2 * i) * 512), 16, 0, 0);
      __builtin_amdgcn_s_waitcnt((7 << 4) | (0xF << 8));  // vmcnt(0): this wave's copies landed
      __syncthreads();
    }
    if (wr == h) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int rl = i * 32 + 8 * (v >> 2) + 4 * fh + (v & 3);
            const int r = 64 * h + rl, c = wc * 64 + j * 32 + fr;
            if (diag_tile && r > c) continue;  // filled from the upper triangle below
            const int64_t gr = r0 + r, gc = c0 + c;
            float x = d.alpha * acc[i][j][v];
            if (E) x += d.beta * tl[rl * kShTile + c];
            if (gr == gc) x += d.diag;
            C[gr * d.ldc + gc] = x;
            acc[i][j][v] = x;
            if (gr < d.valid && gc < d.valid) {
              const float dv = fabsf(x - (gr == gc ? 1.0f : 0.0f));
              res = (dv > res || dv != dv) ? dv : res;  // keeps a NaN
            }
          }
    }
    if (d.sym) {
      if (E) __syncthreads();  // E's LDS reads are done
      if (wr == h) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int rl = i * 32 + 8 * (v >> 2) + 4 * fh + (v & 3);
              const int c = wc * 64 + j * 32 + fr;
              tl[rl * kShTile + (c ^ rl)] = acc[i][j][v];
            }
      }
      __syncthreads();
      const int r = 64 * h + lane;
#pragma unroll 4
      for (int it = 0; it < 32; ++it) {
        const int c = (t >> 6) + 4 * it;
        // position (c, r) of the tile's transpose; on a diagonal tile only below the diagonal
        if (!diag_tile || c > r) C[(c0 + c) * d.ldc + r0 + r] = tl[lane * kShTile + (c ^ lane)];
      }
    }
  }
  if (d.resid_out) {
    // NaN propagates as the largest bit pattern, so a diverged side never counts as converged
    uint32_t rb = __float_as_uint(res);
    if (res != res) rb = 0x7fc00000u;
    for (int o = 32; o > 0; o >>= 1) rb = max(rb, uint32_t(__shfl_xor(int(rb), o)));
    if (lane == 0) atomicMax(reinterpret_cast<unsigned int*>(d.resid_out), rb);
  }
}

// Boundary copy into the padded workspace (optionally transposed as well), 64 x 64 tiles.
__global__ __launch_bounds__(256) void sh_copy_in_kernel(const ShCopyDesc* __restrict__ descs, int count) {
  __shared__ float tt[kShCopyTile][kShCopyTile + 1];
  const int e = find_desc(descs, count, blockIdx.x);
  const ShCopyDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  typedef __attribute__((address_space(1))) uint16_t g_u16;
  const int64_t gc = int64_t(tj) * kShCopyTile + c;
  // a bf16 destination takes the value's upper 16 bits: exact, the values being bf16 numbers
  auto put = [&](void* base, int64_t i, float v) {
    if (d.dst_bf16) ((g_u16*)base)[i] = uint16_t(__float_as_uint(v) >> 16);
    else ((g_f32*)base)[i] = v;
  };
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int r = rr + 4 * i;
    const int64_t gr = int64_t(ti) * kShCopyTile + r;
    const float v = (gr < d.rows && gc < d.cols) ? ld_any(d.src, gr * d.ld_src + gc, d.src_dtype) : 0.0f;
    if (d.dst) put(d.dst, gr * d.ld_dst + gc, v);
    tt[r][c] = v;
  }
  if (d.dstT) {
    __syncthreads();
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
      const int r = rr + 4 * i;  // row of the transposed tile = column of the source tile
      put(d.dstT, (int64_t(tj) * kShCopyTile + r) * d.ld_dstT + int64_t(ti) * kShCopyTile + c, tt[c][r]);
    }
  }
}

// Boundary copy out of the padded workspace into a caller fp32 rows x cols buffer.
__global__ __launch_bounds__(256) void sh_copy_out_kernel(const ShCopyDesc* __restrict__ descs, int count) {
  const int e = find_desc(descs, count, blockIdx.x);
  const ShCopyDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  const g_cf32* src = (const g_cf32*)(d.src);
  g_f32* dst = (g_f32*)(d.dst);
  const int64_t gc = int64_t(tj) * kShCopyTile + c;
  if (gc >= d.cols) return;
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int64_t gr = int64_t(ti) * kShCopyTile + rr + 4 * i;
    if (gr < d.rows) dst[gr * d.ld_dst + gc] = src[gr * d.ld_src + gc];
  }
}

// Sum of squares and trace of one row chunk of a padded statistic, fp64, fixed reduction order.
__global__ __launch_bounds__(256) void sh_norm_kernel(const ShNormDesc* __restrict__ descs, int count) {
  __shared__ double red[2][4];
  const int e = find_desc(descs, count, blockIdx.x);
  const ShNormDesc& d = descs[e];
  const int chunk = blockIdx.x - d.tile_begin;
  const int t = threadIdx.x;
  const int rb = chunk * d.chunk_rows;
  const int re = min(d.rows_pad, rb + d.chunk_rows);
  double ss = 0.0, tr = 0.0;
  for (int r = rb; r < re; ++r) {
    const float* row = d.S + int64_t(r) * d.ld;
    for (int c = t; c < d.rows_pad; c += 256) {
      const double v = row[c];
      ss += v * v;
      if (c == r) tr += v;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    ss += __shfl_xor(ss, o);
    tr += __shfl_xor(tr, o);
  }
  if ((t & 63) == 0) {
    red[0][t >> 6] = ss;
    red[1][t >> 6] = tr;
  }
  __syncthreads();
  if (t == 0) {
    d.partials[2 * chunk] = ((red[0][0] + red[0][1]) + red[0][2]) + red[0][3];
    d.partials[2 * chunk + 1] = ((red[1][0] + red[1][1]) + red[1][2]) + red[1][3];
  }
}

__global__ void sh_scalars_kernel(const ShScalarDesc* __restrict__ descs, int count, double eps,
                                  double eps_rel, int p) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= count) return;
  const ShScalarDesc& d = descs[e];
  double ss = 0.0, tr = 0.0;
  for (int k = 0; k < d.nchunks; ++k) {
    ss += d.partials[2 * k];
    tr += d.partials[2 * k + 1];
  }
  const double rho = eps + eps_rel * sqrt(ss);
  const double n2 = ss + 2.0 * rho * tr + double(d.d) * rho * rho;
  const double z = double(1 + p) / (2.0 * sqrt(n2));
  d.out[0] = float(rho);
  d.out[1] = float(z);
  d.out[2] = float(pow(z, 1.0 / double(p)));
}

// M = z (S + rho I), X = z^(1/p) I (M may alias S).
__global__ __launch_bounds__(256) void sh_init_kernel(const ShInitDesc* __restrict__ descs, int count) {
  const int e = find_desc(descs, count, blockIdx.x);
  const ShInitDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const float rho = d.sc[0], z = d.sc[1], zp = d.sc[2];
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  if (lt == 0 && t < 2) d.resid[t] = t == 0 ? 0.0f : 3.0e38f;
  const int64_t gc = int64_t(tj) * kShCopyTile + c;
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int64_t gr = int64_t(ti) * kShCopyTile + rr + 4 * i;
    const int64_t o = gr * d.ld + gc;
    const bool dg = gr == gc;
    d.M[o] = z * (d.S[o] + (dg ? rho : 0.0f));
    d.X[o] = dg ? zp : 0.0f;
  }
}

__global__ __launch_bounds__(256) void sh_apply_kernel(const ShApplyDesc* __restrict__ descs, int count,
                                                       float decay, float step) {
  const int e = find_desc(descs, count, blockIdx.x);
  const ShApplyDesc& d = descs[e];
  const int lt = blockIdx.x - d.tile_begin;
  const int ti = lt / d.tiles_n, tj = lt - ti * d.tiles_n;
  const int t = threadIdx.x, c = t & 63, rr = t >> 6;
  const int64_t gc = int64_t(tj) * kShCopyTile + c;
  if (gc >= d.n) return;
#pragma unroll 4
  for (int i = 0; i < 16; ++i) {
    const int64_t gr = int64_t(ti) * kShCopyTile + rr + 4 * i;
    if (gr >= d.m) continue;
    const float u = d.U[gr * d.ldu + gc];
    const int64_t o = gr * d.n + gc;
    if (d.param_dtype == kDtBF16) {
      uint16_t* pp = static_cast<uint16_t*>(d.param);
      const float p = __uint_as_float(uint32_t(pp[o]) << 16);
      pp[o] = uint16_t(pack_bf16x2(p * decay - step * u, 0.0f) & 0xffffu);
    } else {
      float* pp = static_cast<float*>(d.param);
      pp[o] = pp[o] * decay - step * u;
    }
    if (d.update_out) d.update_out[o] = u;
  }
}

}  // namespace

hipError_t launch_sh_gemm(const ShGemmDesc* d, int count, int total_tiles, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(sh_gemm_kernel, dim3(total_tiles), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_sh_copy(const ShCopyDesc* d, int count, int total_tiles, int dir, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  if (dir == 0)
    hipLaunchKernelGGL(sh_copy_in_kernel, dim3(total_tiles), dim3(256), 0, st, d, count);
  else
    hipLaunchKernelGGL(sh_copy_out_kernel, dim3(total_tiles), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_sh_norm(const ShNormDesc* d, int count, int total_blocks, hipStream_t st) {
  if (total_blocks <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(sh_norm_kernel, dim3(total_blocks), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_sh_scalars(const ShScalarDesc* d, int count, double eps, double eps_rel, int p,
                             hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(sh_scalars_kernel, dim3((count + 63) / 64), dim3(64), 0, st, d, count, eps,
                     eps_rel, p);
  return hipGetLastError();
}

hipError_t launch_sh_init(const ShInitDesc* d, int count, int total_tiles, hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(sh_init_kernel, dim3(total_tiles), dim3(256), 0, st, d, count);
  return hipGetLastError();
}

hipError_t launch_sh_apply(const ShApplyDesc* d, int count, int total_tiles, float decay, float step,
                           hipStream_t st) {
  if (total_tiles <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(sh_apply_kernel, dim3(total_tiles), dim3(256), 0, st, d, count, decay, step);
  return hipGetLastError();
}

}  // namespace mfsdp
