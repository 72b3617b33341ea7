// Newton-Schulz products on gfx950.
//
// Every product of the quintic step is computed as one grouped "NT" GEMM
//     C = alpha * P Q^T + beta * E        (P: M x K, Q: N x K, both K-contiguous, panel blocked)
// over all matrices of the owner in one launch (one problem per matrix). Symmetric products
// (A = X X^T and B' = c A A + b A + a I) compute only the tiles on and above the diagonal and
// store each off-diagonal tile twice (as is and transposed).
//
// bf16 path: a persistent grid of one workgroup per CU (8 waves) walks a host-built tile schedule
// (TileRef); each 256 x 256 output tile is 2 x 4 waves of 128 x 64, as 4 x 2 blocks of
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation. K advances 32 elements per step through a
// five-stage LDS ring filled by direct global->LDS loads; the next tile's first loads overlap the
// current tile's epilogue. The Gram and square products of a small share run the same kernel on
// 128 x 128 tiles (2 x 2 waves of 64 x 64, two workgroups per CU), four times the tiles.
// fp32 path: 64 x 64 tiles on the fp32 MFMA (v_mfma_f32_32x32x2f32).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "mfsdp_internal.h"

namespace mfsdp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
// global-address-space element types (pointers derived from these give global_* instructions)
typedef __attribute__((address_space(1))) uint16_t gu16;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) u32x2 gu2;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 gu4;

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>), unrolled by construction.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// DPP quad permutations: lane i of each group of 4 reads lane i ^ 1 (quad_perm [1,0,3,2]) or
// lane i ^ 2 (quad_perm [2,3,0,1]).
__device__ __forceinline__ float dpp_quad_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_quad_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));
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

// Fused parameter update for 4 consecutive elements (pr, pc .. pc + 3) of the stored m x n
// parameter, pc a multiple of 4: p <- p (1 - lr wd) - lr f O (mode 0, optionally also writing O to
// update_out), or p <- O (mode 1, standalone NS output). Elements outside m x n are skipped.
__device__ __forceinline__ void apply4(const ApplyDesc& a, int64_t pr, int64_t pc, float o0,
                                       float o1, float o2, float o3) {
  typedef __attribute__((address_space(1))) float gf32;
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) f32x4 gf4;
  const int64_t m = a.m, n = a.n;
  if (pr >= m || pc >= n) return;
  const int64_t idx = pr * n + pc;
  const float o[4] = {o0, o1, o2, o3};
  const bool bf = a.param_dtype == kDtBF16;
  if ((n & 3) == 0) {  // then pc + 3 < n, and the 4 elements are 8 / 16-byte aligned
    float r[4] = {o0, o1, o2, o3};
    if (a.mode == 0) {
      float p[4];
      if (bf) {
        const u32x2 w = *(const gu2*)((const gu16*)a.param + idx);
        p[0] = __uint_as_float(w.x << 16); p[1] = __uint_as_float(w.x & 0xffff0000u);
        p[2] = __uint_as_float(w.y << 16); p[3] = __uint_as_float(w.y & 0xffff0000u);
      } else {
        const f32x4 w = *(const gf4*)((const gf32*)a.param + idx);
        p[0] = w.x; p[1] = w.y; p[2] = w.z; p[3] = w.w;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) r[k] = p[k] * a.decay - a.step * o[k];
      if (a.update_out) *(gf4*)((gf32*)a.update_out + idx) = f32x4{o0, o1, o2, o3};
    }
    if (bf) *(gu2*)((gu16*)a.param + idx) = u32x2{pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3])};
    else *(gf4*)((gf32*)a.param + idx) = f32x4{r[0], r[1], r[2], r[3]};
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (pc + k >= n) break;
      float r = o[k];
      if (a.mode == 0) {
        const float p = bf ? __uint_as_float(uint32_t(((const gu16*)a.param)[idx + k]) << 16)
                           : ((const gf32*)a.param)[idx + k];
        r = p * a.decay - a.step * o[k];
        if (a.update_out) ((gf32*)a.update_out)[idx + k] = o[k];
      }
      if (bf) ((gu16*)a.param)[idx + k] = uint16_t(pack_bf16x2(r, 0.0f));
      else ((gf32*)a.param)[idx + k] = r;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// bf16 MFMA kernel
//
// Main loop: K in steps of 32 elements. A stage holds the P rows (TB x 32 bf16: 16 KiB on 256 x 256
// tiles) followed by the Q rows of one K step. Stages are filled by direct global->LDS loads
// (global_load_lds_dwordx4: each wave instruction writes 64 x 16 B = 1 KiB of LDS contiguously),
// so no registers or ds_write instructions carry the tiles. One workgroup barrier per K step kt,
// placed between its two 16-wide K slices: before it every wave that issues loads waits (explicit
// vmcnt) for its loads of step kt + 1; after it the loads of step kt + NSTAGE - 1 are issued into
// the stage of step kt - 1 (whose last fragments were consumed by MFMAs issued before the
// barrier), and the first fragments of step kt + 1 are read while the second slice of step kt is
// multiplied. Steps kt + 2 .. kt + NSTAGE - 1 are in flight meanwhile.
//
// LDS row layout: 64 B per row = four 16-B chunks; chunk c of row r is stored in slot c ^ g(r)
// with g(r) = (r1 ^ r3) | r2 << 1 (bits of r). Groups of 8 (or 16) consecutive rows read by one
// ds_read_b128 cycle then hit distinct banks for 32 (or 64) banks of 4 B.
constexpr int BT = 256;                      // output tile (both sides) of the full-size kernel
constexpr int BKE = 32;                      // K elements per stage
constexpr int ROWB = BKE * 2;                // bytes per staged row (64)
constexpr int NSTAGE = 5;                    // 160 KiB of LDS (80 KiB on 128 x 128 tiles)

typedef __attribute__((address_space(3))) uint8_t lds_byte;

__device__ __forceinline__ int swz(int r) { return ((r >> 1 ^ r >> 3) & 1) | (((r >> 2) & 1) << 1); }

// s_waitcnt with only vmcnt constrained (expcnt and lgkmcnt left at their maxima).
#define MFSDP_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (7 << 4) | (0xF << 8))
// s_waitcnt lgkmcnt(0) only (LDS writes done before a barrier; outstanding global loads and stores
// are not waited for)
#define MFSDP_WAIT_LGKM0() __builtin_amdgcn_s_waitcnt(0xF | (7 << 4) | (0 << 8) | (3 << 14))

constexpr int kGemmWaves = 8;  // waves per workgroup of the bf16 kernel on 256 x 256 tiles
constexpr int kGemmWavesSmall = 4;  // and on 128 x 128 tiles (two workgroups per CU)
// NW waves per workgroup arranged WM x WN over the TB x TB tile; each wave owns
// (TB / WM) x (TB / WN) outputs as MI x NI blocks of 32 x 32. Two waves share each SIMD (8 waves
// of one workgroup, or 4 of each of two), so one can issue while the other waits.
template <int NW, int TB>
struct WaveGrid {
  static constexpr int WM = 2;
  static constexpr int WN = NW / 2;
  static constexpr int MI = TB / (WM * 32);
  static constexpr int NI = TB / (WN * 32);
  static constexpr int LOADS = 2 * TB / kBlkRows / NW;  // DMA instructions per thread per stage
  static constexpr int STAGE = 2 * TB * ROWB;           // bytes per stage: P rows, then Q rows
  static constexpr int SLOTS = TB == BT ? kGemmSlots : 2 * kGemmSlots;  // workgroups per XCD
};

// Per-tile state of the persistent kernel: operand sources of the DMA and the tile coordinates.
struct TileCtx {
  const GemmDesc* d;
  int bi, bj, nk, ks;
  const uint16_t* psrc;
  const uint16_t* qsrc;
  int64_t pstep, qstep;
};

// Product kinds of one NS step (one launch each); the epilogue is specialised per kind.
constexpr int kProdGram = 0;    // A = X X^T: symmetric, mirror stores
constexpr int kProdSquare = 1;  // B' = c A A + b A + a I: symmetric, addend E = A, diagonal term
constexpr int kProdUpdate = 2;  // X' = B' X: stores X' and X'^T
constexpr int kProdApply = 3;   // the last X' = B' X, applying the parameter update (or writing the
                                // standalone NS output) instead of storing X'; its own instantiation,
                                // so that each update kernel carries only its own epilogue

// (ca, cb, cc): this NS step's coefficients; the square product uses them as diagonal term, addend
// factor and product factor (B' = cc A A + cb A + ca I).
template <int NW, int TB, int PK>
__global__ __launch_bounds__(NW * 64, TB == BT ? 1 : 2) void gemm_bf16_kernel(
    const GemmDesc* __restrict__ descs, const TileRef* __restrict__ sched, int ngroups, int parity,
    int first, int last, float ca, float cb, float cc) {
  using WG = WaveGrid<NW, TB>;
  constexpr int MI = WG::MI, NI = WG::NI, LOADS = WG::LOADS, STAGE_BYTES = WG::STAGE;
  // The first DW waves issue all of a stage's global->LDS loads (DLOADS each). With 8 waves that is
  // the first four, one per SIMD: each SIMD then runs one wave that issues loads and one that
  // never waits on their issue and keeps multiplying meanwhile.
  constexpr int DW = NW == 8 ? 4 : NW;
  constexpr int DLOADS = LOADS * NW / DW;
  constexpr int PL = DLOADS / 2;       // DMA instructions for P (and for Q) per issuing thread
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NSTAGE * STAGE_BYTES];

  const int xcd = blockIdx.x % kGemmXcds, slot = blockIdx.x / kGemmXcds;
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  const int wm = w / WG::WN, wn = w % WG::WN;
  // DMA mapping: instruction c of issuing wave w covers staged rows j * 16 + lane / 4 with
  // j = c * DW + w; j < TB / 16 are P rows, the others the rows j - TB / 16 of Q. Lane slot =
  // lane % 4 holds global chunk slot ^ swz(row) (swz depends on row % 16 = lane / 4 only).
  const bool issuer = w < DW;
  const int drow = (w % DW) * 16 + (lane >> 2);
  const int dchunk = (lane & 3) ^ swz(lane >> 2);
  const int dma_wave_off = (w % DW) * 1024;  // + c * DW * 1024 within a stage

  // next non-idle tile of this workgroup at or after group g (g advances by kGemmXcds)
  auto next_tile = [&](int& g, TileCtx& c) -> bool {
    for (; g < ngroups; g += kGemmXcds) {
      const TileRef r = sched[g * WG::SLOTS + slot];
      if (r.e < 0) continue;
      const GemmDesc& dd = descs[r.e];
      c.d = &dd;
      c.bi = r.bi;
      c.bj = r.bj;
      c.ks = r.ks;
      // a split Gram tile covers K range ks of nks (each range a whole number of 16 x 32 blocks:
      // it starts nk * ks blocks further along every panel)
      const int nks = (PK == kProdGram && dd.nks > 1) ? dd.nks : 1;
      c.nk = dd.K / BKE / nks;
      const int64_t k0 = int64_t(c.nk) * (nks > 1 ? r.ks : 0) * (kBlkRows * BKE);
      const uint16_t* P = static_cast<const uint16_t*>(dd.P[parity]);
      const uint16_t* Q = static_cast<const uint16_t*>(dd.Q[parity]);
      c.psrc = P + blk_index(int64_t(c.bi) * TB + drow, dchunk * 8, dd.ldp) + k0;
      c.qsrc = Q + blk_index(int64_t(c.bj) * TB + drow, dchunk * 8, dd.ldq) + k0;
      c.pstep = int64_t(DW * kBlkRows) * dd.ldp;  // DW row panels further down
      c.qstep = int64_t(DW * kBlkRows) * dd.ldq;
      return true;
    }
    return false;
  };
  auto issue = [&](const TileCtx& c, int kt, int stage) {
    const int64_t koff = int64_t(kt) * (kBlkRows * BKE);  // next 16 x 32 block of the panel
    lds_byte* sb = (lds_byte*)(smem + stage * STAGE_BYTES + dma_wave_off);
#pragma unroll
    for (int i = 0; i < PL; ++i)
      __builtin_amdgcn_global_load_lds(c.psrc + i * c.pstep + koff, sb + i * DW * 1024, 16, 0, 0);
#pragma unroll
    for (int i = 0; i < PL; ++i)
      __builtin_amdgcn_global_load_lds(c.qsrc + i * c.qstep + koff, sb + TB * ROWB + i * DW * 1024, 16, 0,
                                       0);
  };
  // steps 0 .. NSTAGE-2 of a tile into stages 0 .. NSTAGE-2 (steps past the end are clamped to the
  // last one: in-bounds reloads into stages nobody reads)
  auto prologue = [&](const TileCtx& c) {
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s) issue(c, s < c.nk ? s : c.nk - 1, s);
  };

  // fragment reads: row (base + lane % 32), chunk q = 2 kk + lane / 32 at slot q ^ swz(lane % 32)
  const int frow = lane & 31, fhalf = lane >> 5;
  const int pbase = (wm * (MI * 32) + frow) * ROWB;
  const int qbase = (TB + wn * (NI * 32) + frow) * ROWB;
  const int slot0 = ((0 + fhalf) ^ swz(frow)) * 16;
  const int slot1 = ((2 + fhalf) ^ swz(frow)) * 16;
  constexpr int NMF = MI * NI;      // MFMAs per 16-wide K slice
  constexpr int NRD = MI + NI;      // fragment reads per slice

  int g = xcd;
  TileCtx cur;
  if (!next_tile(g, cur)) return;
  if (issuer) prologue(cur);
  while (true) {
    g += kGemmXcds;
    TileCtx nxt;
    const bool has_next = next_tile(g, nxt);

    f32x16_t acc[MI][NI];
#pragma unroll
    for (int a = 0; a < MI; ++a)
#pragma unroll
      for (int b = 0; b < NI; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

    bf16x8_t pf0[MI], qf0[NI], pf1[MI], qf1[NI];
    auto read_frags = [&](const uint8_t* sb, int sl, bf16x8_t* pf, bf16x8_t* qf) {
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
        pf[mi] = *reinterpret_cast<const bf16x8_t*>(sb + pbase + mi * 32 * ROWB + sl);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        qf[ni] = *reinterpret_cast<const bf16x8_t*>(sb + qbase + ni * 32 * ROWB + sl);
    };
    auto mfma_slice = [&](const bf16x8_t* pf, const bf16x8_t* qf) {
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ni], pf[mi], acc[mi][ni], 0, 0, 0);
    };

    // Main loop. Outstanding vector-memory operations of an issuing wave at this point: this tile's
    // prologue loads, then the previous tile's epilogue stores. Loads complete in order among
    // themselves, so "at most (NSTAGE - 2) * DLOADS outstanding" implies step 0 has landed whether
    // or not stores retire in order with loads (if they do, this waits a little longer than needed).
    // The other waves have no loads to wait for: the barrier after the issuers' wait covers them.
    auto main_loop = [&](auto issue_c) {
      constexpr bool ISS = decltype(issue_c)::value;
      constexpr int L = ISS ? DLOADS : 0;  // DMA instructions of this wave per K step
      const int nk = cur.nk, last_kt = nk - 1;
      if constexpr (ISS) MFSDP_WAIT_VMCNT((NSTAGE - 2) * DLOADS);
      __builtin_amdgcn_s_barrier();
      read_frags(smem, slot0, pf0, qf0);
      int cs = 0, ns = 1, fs = NSTAGE - 1;  // stages of steps kt, kt + 1 and of step kt + NSTAGE - 1
      for (int kt = 0; kt < nk; ++kt) {
        const uint8_t* sb = smem + cs * STAGE_BYTES;
        read_frags(sb, slot1, pf1, qf1);
        mfma_slice(pf0, qf0);
        // scheduling: pairs of 1 MFMA + 1 fragment read, then the remaining MFMAs
        static_assert(NMF >= NRD && NMF >= DLOADS, "slice schedule assumes more MFMAs than reads");
#pragma unroll
        for (int i = 0; i < NRD; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // 1 LDS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NMF - NRD, 0);
        // step kt + 1 must have landed (steps kt + 2 .. kt + NSTAGE - 2 may still be in flight)
        if constexpr (ISS) MFSDP_WAIT_VMCNT((NSTAGE - 3) * DLOADS);
        __builtin_amdgcn_s_barrier();
        if constexpr (ISS) {
          const int kload = kt + NSTAGE - 1;
          issue(cur, kload < nk ? kload : last_kt, fs);
        }
        read_frags(smem + ns * STAGE_BYTES, slot0, pf0, qf0);
        mfma_slice(pf1, qf1);
        if constexpr (DW == NW) {
          // scheduling: pairs of 1 MFMA + 1 DMA issue, then pairs of 1 MFMA + 1 fragment read while
          // MFMAs last, then the remaining reads
          constexpr int PAIRED = (NMF - L < NRD) ? NMF - L : NRD;
#pragma unroll
          for (int i = 0; i < L; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // 1 VMEM (DMA) issue
          }
#pragma unroll
          for (int i = 0; i < PAIRED; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          if constexpr (NRD > PAIRED) __builtin_amdgcn_sched_group_barrier(0x100, NRD - PAIRED, 0);
          if constexpr (NMF - L > PAIRED) __builtin_amdgcn_sched_group_barrier(0x008, NMF - L - PAIRED, 0);
        } else {
          // scheduling: each MFMA followed by this wave's next DMA issue and next fragment read,
          // while there are any
#pragma unroll
          for (int i = 0; i < NMF; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i < L) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            if (i < NRD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
        }
        cs = ns;
        ns = (ns + 1 == NSTAGE) ? 0 : ns + 1;
        fs = (fs + 1 == NSTAGE) ? 0 : fs + 1;
      }
    };
    if (issuer)
      main_loop(std::true_type{});
    else
      main_loop(std::false_type{});
    // The clamped tail loads of this tile must land before the next tile's prologue reuses the
    // stages, and every wave must be done reading LDS (its last fragments were consumed by MFMAs).
    MFSDP_WAIT_VMCNT(0);
    __builtin_amdgcn_s_barrier();
    if (has_next && issuer) prologue(nxt);  // overlaps the epilogue below (it leaves stage NSTAGE-1 free)

    // Epilogue (global-address-space accesses: flat ones would also hold lgkmcnt, which the next
    // tile's LDS reads wait on). acc[mi][ni] holds D[j][i] = C[i][j] with i = i0 + lane % 32 and
    // j = j0 + 8 g + 4 (lane / 32) + t for element v = 4 g + t: each lane has 4 consecutive columns
    // of one row per group g (one 8-byte row-major store). For the transposed stores (X'^T, and the
    // mirrored tile of a symmetric product) the 4 x 4 blocks held by lane quads are transposed with
    // two DPP exchanges, so each lane then holds 4 consecutive rows of one column (again one 8-byte
    // store).
    const GemmDesc& dd = *cur.d;
    const int bi = cur.bi, bj = cur.bj;
    if constexpr (PK == kProdGram) {
      if (dd.nks > 1) {
        // split contraction: this K range's fp32 partial tile, row-major, 16-byte stores straight
        // from the accumulators (each lane: 4 consecutive columns of one row per group); the
        // second pass forms A
        typedef float f32x4s __attribute__((ext_vector_type(4)));
        typedef __attribute__((address_space(1))) f32x4s gf4s;
        float* part = dd.part + (int64_t(upper_index(bi, bj, dd.tiles_m)) * dd.nks + cur.ks) * (TB * TB);
        static_for<MI>([&](auto mi_c) {
          constexpr int mi = decltype(mi_c)::value;
          const int il = wm * (MI * 32) + mi * 32 + frow;
          static_for<NI>([&](auto ni_c) {
            constexpr int ni = decltype(ni_c)::value;
            static_for<4>([&](auto gg_c) {
              constexpr int gg = decltype(gg_c)::value;
              const int jl = wn * (NI * 32) + ni * 32 + gg * 8 + fhalf * 4;
              *(gf4s*)(part + il * TB + jl) = f32x4s{acc[mi][ni][4 * gg], acc[mi][ni][4 * gg + 1],
                                                     acc[mi][ni][4 * gg + 2], acc[mi][ni][4 * gg + 3]};
            });
          });
        });
        if (!has_next) break;
        cur = nxt;
        continue;
      }
    }
    const float alpha = PK == kProdSquare ? cc : dd.alpha * (first ? scale_pow(dd.scale, dd.alpha_scale_pow) : 1.0f);
    const float beta = PK == kProdSquare ? cb : dd.beta * (first ? scale_pow(dd.scale, dd.beta_scale_pow) : 1.0f);
    const float diag = (PK == kProdSquare && bi == bj) ? ca : 0.0f;
    const gu16* E = (const gu16*)dd.E[parity];
    gu16* C = (gu16*)dd.C[parity];
    gu16* CT = (gu16*)dd.CT[parity];
    const ApplyDesc* fa = PK == kProdApply ? dd.fused : nullptr;  // set by the host for this kind
    if (last) {
      if (!dd.last_c || fa) C = nullptr;
      if (!dd.last_ct || fa) CT = nullptr;
    }
    // fused update of a tall parameter: it is X'^T, so it takes the transposed values
    const bool fa_t = fa && fa->m > fa->n;
    // transposed destination: the mirror tile of a symmetric product, or X'^T
    gu16* TD = (dd.sym && bi != bj && C) ? C : CT;
    const int64_t ldtd = (TD == C) ? dd.ldc : dd.ldct;
    const int64_t lde = dd.lde, ldc = dd.ldc;
    const int q = lane & 3;
    const bool q_odd = q & 1, q_hi = q & 2;
    // 4 x 4 transpose within each lane quad: afterwards lane q holds column j + q at rows iq .. iq + 3
    auto quad_transpose = [&](float& v0, float& v1, float& v2, float& v3) {
      // exchange across lane ^ 1: even lanes take the partner's elements 0, 2 as their 1, 3
      {
        const float x0 = q_odd ? v0 : v1, x1 = q_odd ? v2 : v3;
        const float y0 = dpp_quad_xor1(x0), y1 = dpp_quad_xor1(x1);
        if (q_odd) { v0 = y0; v2 = y1; } else { v1 = y0; v3 = y1; }
      }
      // exchange across lane ^ 2: low lanes take the partner's elements 0, 1 as their 2, 3
      {
        const float x0 = q_hi ? v0 : v2, x1 = q_hi ? v1 : v3;
        const float y0 = dpp_quad_xor2(x0), y1 = dpp_quad_xor2(x1);
        if (q_hi) { v0 = y0; v1 = y1; } else { v2 = y0; v3 = y1; }
      }
    };
    if (PK == kProdApply && TB == BT && fa->param_dtype == kDtBF16 && (fa->n & 7) == 0) {
      // Fused update of a bf16 parameter with n % 8 == 0, staged through the LDS stage the next
      // tile's prologue leaves free (32 KiB of fp32 per round), so that each wave reads and writes
      // whole parameter row segments with 16-byte lanes: p <- p (1 - lr wd) - lr f O in fp32 from
      // the unrounded O, one rounding to bf16; eight rounds per tile, each reading its parameter
      // words before its LDS exchange. A wide parameter's rows are tile rows (rounds of 64 tile rows
      // x 128 columns, 256-byte row segments); a tall parameter's rows are tile columns (rounds of
      // one 32 x 32 block per wave, 64-byte row pieces), so that every wave's accumulators die
      // round by round. 16-byte slots are XOR-swizzled per row so that the writes and the 16-lane
      // reads hit 16 distinct bank groups (checked on the CPU with a bank model).
      typedef float f32x4 __attribute__((ext_vector_type(4)));
      typedef __attribute__((address_space(1))) float gf32;
      typedef __attribute__((address_space(1))) f32x4 gf4;
      typedef __attribute__((address_space(3))) f32x4 lf4;
      lds_byte* slab = (lds_byte*)(smem + (NSTAGE - 1) * STAGE_BYTES);
      int ln = lane;
      asm volatile("" : "+v"(ln));
      const int frow = ln & 31, fhalf = ln >> 5, qd = ln & 3;
      const int64_t fm = fa->m, fn = fa->n;
      const float decay = fa->decay, stp = fa->step;
      const int mode = fa->mode;
      gu16* prm = (gu16*)fa->param;
      gf32* uo = (gf32*)fa->update_out;
      // Rounds R = 0 .. 7 (wide: block row mi = R / 2, column half h = R % 2; tall: block (mi, ni) =
      // (R / NI, R % NI) of every wave).
      // Lane coordinates of its two 8-element parameter pieces (it = 0, 1) in round R.
      auto coords = [&](int R, int it, int64_t& pr, int64_t& pc) {
        if (!fa_t) {
          const int sr = w * 8 + it * 4 + (ln >> 4);
          const int trow = (sr >> 5) * (MI * 32) + (R >> 1) * 32 + (sr & 31);
          pr = int64_t(bi) * BT + trow;
          pc = int64_t(bj) * BT + (R & 1) * 128 + (ln & 15) * 8;
        } else {
          // round (mi, ni) = (R / NI, R % NI); parameter row = tile column, columns = tile rows
          const int jc = w * 16 + it * 8 + (ln >> 3), p = (ln >> 2) & 1, c4 = ln & 3;
          pr = int64_t(bj) * BT + (jc >> 5) * (NI * 32) + (R % NI) * 32 + (jc & 31);
          pc = int64_t(bi) * BT + p * (MI * 32) + (R / NI) * 32 + c4 * 8;
        }
      };
      // the parameter words of round R, loaded before the round's LDS exchange so that it covers
      // their latency (the read is the one dependent HBM access of this epilogue; the other
      // epilogues only store)
      auto load_round = [&](int R, u32x4* dst) {
#pragma unroll
        for (int it = 0; it < 2; ++it) {
          int64_t pr, pc;
          coords(R, it, pr, pc);
          dst[it] = u32x4{0u, 0u, 0u, 0u};
          if (mode == 0 && pr < fm && pc < fn) dst[it] = *(const gu4*)(prm + pr * fn + pc);
        }
      };
      // parameter elements (pr, pc .. pc + 7) from the fp32 values o0, o1 of O and the old words pw
      auto update8 = [&](int64_t pr, int64_t pc, f32x4 o0, f32x4 o1, u32x4 pw) {
        if (pr >= fm || pc >= fn) return;
        const int64_t idx = pr * fn + pc;
        float r[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
        if (mode == 0) {
          const uint32_t wv[4] = {pw.x, pw.y, pw.z, pw.w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            r[2 * k] = __uint_as_float(wv[k] << 16) * decay - stp * r[2 * k];
            r[2 * k + 1] = __uint_as_float(wv[k] & 0xffff0000u) * decay - stp * r[2 * k + 1];
          }
          if (uo) {
            *(gf4*)(uo + idx) = o0;
            *(gf4*)(uo + idx + 4) = o1;
          }
        }
        *(gu4*)(prm + idx) = u32x4{pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]),
                                   pack_bf16x2(r[4], r[5]), pack_bf16x2(r[6], r[7])};
      };
      // 16-byte slot swizzles of the two slab layouts (bijective within a row; conflict-free writes
      // and 16-lane reads in a CPU bank model)
      auto wsw = [](int row, int slot) { return (slot ^ (row & 31)) ^ ((slot >> 4) & 1); };
      auto tsw = [](int jc, int slot) { return (slot ^ ((jc & 3) << 2) ^ ((jc & 1) * 3)) & 15; };
      // second half of a round (the writes are done): exchange O through the slab, update
      auto finish_round = [&](int R, const u32x4* pw, auto read_o) {
        MFSDP_WAIT_LGKM0();
        __builtin_amdgcn_s_barrier();
#pragma unroll
        for (int it = 0; it < 2; ++it) {
          f32x4 o0, o1;
          read_o(it, o0, o1);
          int64_t pr, pc;
          coords(R, it, pr, pc);
          update8(pr, pc, o0, o1, pw[it]);
        }
        __builtin_amdgcn_s_barrier();  // slab reads done before the next round writes
      };
      if (!fa_t) {
        // slab [64 rows][32 slots of 16 B]; round (mi, h): tile rows wm * 128 + mi * 32 + [0, 32)
        // of both wave rows, tile columns h * 128 + [0, 128), written by the waves of that half
        static_for<MI>([&](auto mi_c) {
          constexpr int mi = decltype(mi_c)::value;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            u32x4 pw[2];
            load_round(mi * 2 + h, pw);
            if ((wn >> 1) == h) {
              const int sr = wm * 32 + frow;
              static_for<NI>([&](auto ni_c) {
                constexpr int ni = decltype(ni_c)::value;
                static_for<4>([&](auto gg_c) {
                  constexpr int gg = decltype(gg_c)::value;
                  const int slot = (wn & 1) * 16 + ni * 8 + gg * 2 + fhalf;
                  *(lf4*)(slab + sr * 512 + wsw(sr, slot) * 16) =
                      f32x4{alpha * acc[mi][ni][4 * gg], alpha * acc[mi][ni][4 * gg + 1],
                            alpha * acc[mi][ni][4 * gg + 2], alpha * acc[mi][ni][4 * gg + 3]};
                });
              });
            }
            finish_round(mi * 2 + h, pw, [&](int it, f32x4& o0, f32x4& o1) {
              const int sr = w * 8 + it * 4 + (ln >> 4), c = ln & 15;
              o0 = *(lf4*)(slab + sr * 512 + wsw(sr, 2 * c) * 16);
              o1 = *(lf4*)(slab + sr * 512 + wsw(sr, 2 * c + 1) * 16);
            });
          }
        });
      } else {
        // slab [128 tile columns][16 slots of 16 B, 4 tile rows each]; round (mi, ni): every
        // wave's block (mi, ni), i.e. tile rows wm * 128 + mi * 32 + [0, 32) and tile columns
        // wn * 64 + ni * 32 + [0, 32), written after a quad transpose; each of the 128 parameter
        // rows (tile columns) then takes two 32-element pieces (one per wave row)
        static_for<MI>([&](auto mi_c) {
          constexpr int mi = decltype(mi_c)::value;
          static_for<NI>([&](auto ni_c) {
            constexpr int ni = decltype(ni_c)::value;
            u32x4 pw[2];
            load_round(mi * NI + ni, pw);
            static_for<4>([&](auto gg_c) {
              constexpr int gg = decltype(gg_c)::value;
              float v0 = alpha * acc[mi][ni][4 * gg + 0];
              float v1 = alpha * acc[mi][ni][4 * gg + 1];
              float v2 = alpha * acc[mi][ni][4 * gg + 2];
              float v3 = alpha * acc[mi][ni][4 * gg + 3];
              quad_transpose(v0, v1, v2, v3);  // lane qd: column + qd at tile rows iq .. iq + 3
              const int jc = wn * 32 + gg * 8 + fhalf * 4 + qd;
              *(lf4*)(slab + jc * 256 + tsw(jc, wm * 8 + (frow >> 2)) * 16) = f32x4{v0, v1, v2, v3};
            });
            finish_round(mi * NI + ni, pw, [&](int it, f32x4& o0, f32x4& o1) {
              const int jc = w * 16 + it * 8 + (ln >> 3), p = (ln >> 2) & 1, c4 = ln & 3;
              o0 = *(lf4*)(slab + jc * 256 + tsw(jc, p * 8 + c4 * 2) * 16);
              o1 = *(lf4*)(slab + jc * 256 + tsw(jc, p * 8 + c4 * 2 + 1) * 16);
            });
          });
        });
      }
      if (!has_next) break;
      cur = nxt;
      continue;
    }
    if constexpr (PK != kProdApply) {
      // Staged epilogue. The output tile leaves through the LDS stage the next tile's prologue does
      // not use, one 64-row slab (32 rows of each wave row) per round: the waves write their
      // values into the slab in the global panel-blocked layout, then each wave stores whole 1 KiB
      // blocks with 16-byte lanes, read back as they are (C) or with transposing LDS reads (the
      // transposed output: X'^T, or the mirror tile of a symmetric product). Per element this
      // costs a scale, a conversion and a share of one LDS write; scattered 8-byte stores straight
      // from the accumulators, and DPP transposes, measured much slower.
      lds_byte* slab = (lds_byte*)(smem + (NSTAGE - 1) * STAGE_BYTES);
      typedef __attribute__((address_space(3))) u32x2 l2x;
      typedef __attribute__((address_space(3))) u32x4 l4x;
      typedef __attribute__((address_space(3))) bf16x4_t lbf4;
      // The lane index passes through an empty asm so that the lane-dependent offsets below are
      // formed here, per tile: hoisted out of the tile loop they would stay live through the main
      // loop and push it into spilling.
      int ln = lane;
      asm volatile("" : "+v"(ln));
      const int frow = ln & 31, fhalf = ln >> 5;
      // slab byte offset of (row sr, column c): 16 x 32 blocks (block (sr / 16, c / 32) at
      // 1 KiB * (8 (sr / 16) + c / 32)), 64-byte block rows whose 16-byte chunks are swizzled by
      // swz(row % 16)
      auto slab_off = [](int sr, int c) -> int {
        return (((sr >> 4) * (TB / 32) + (c >> 5)) << 10) + ((sr & 15) << 6) +
               ((((c & 31) >> 3) ^ swz(sr & 15)) << 4) + ((c & 7) << 1);
      };
      // this lane's slab writes: row wm * 32 + frow, columns wn * 64 + ni * 32 + gg * 8 + fhalf * 4
      const int sr_w = wm * 32 + frow;
      const int wr_base = slab_off(sr_w, wn * (NI * 32) + fhalf * 4);  // ni = gg = 0
      const int wr_sw = swz(sr_w & 15);
      // C block stores: lane = 4 row_in + ch holds row row_in, 16-byte chunk ch of a block
      const int row_in = ln >> 2, ch = ln & 3;
      const int rd_off = (row_in << 6) + ((ch ^ swz(row_in)) << 4);
      // transposed block stores: lane = 16 g + il holds row il (a tile column) and columns
      // 8 g .. 8 g + 7 (tile rows) of a 16 x 32 block of the transposed tile, from two
      // ds_read_b64_tr_b16 of slab rows 8 g + r (+ 4), r = 0..3, columns 4 c .. 4 c + 3 (lane of
      // the 16-lane group = 4 r + c)
      const int tg = ln >> 4, til = ln & 15, tr_r = (ln >> 2) & 3, tr_c = ln & 3;
      constexpr int BPW = 4 * (TB / 32) / NW;  // blocks of a slab (64 rows) stored per wave
      const float* dscale = dd.scale;
      (void)dscale;
      const int ldc32 = int(ldc), ldtd32 = int(ldtd);
      gu16* Ct = C ? C + blk_index(int64_t(bi) * TB, int64_t(bj) * TB, ldc) : nullptr;
      gu16* Tt = TD ? TD + blk_index(int64_t(bj) * TB, int64_t(bi) * TB, ldtd) : nullptr;
      const gu16* Et = nullptr;
      int lde32 = 0;
      if constexpr (PK == kProdSquare) {
        Et = E + blk_index(int64_t(bi) * TB, int64_t(bj) * TB, dd.lde);
        lde32 = int(dd.lde);
      }
      // values of round mi into the slab; DIAG: this is a diagonal tile of the square product
      // The square product's addend E = A for round mi: each lane's 4-element pieces, loaded one
      // round ahead of their use (double-buffered by round parity) so that their latency is covered
      // by the previous round's exchange instead of stalling each round.
      u32x2 ev[2][NI][4];
      auto load_e = [&](auto mi_c) {
        constexpr int mi = decltype(mi_c)::value;
        const int il = wm * (MI * 32) + mi * 32 + frow;
        static_for<NI>([&](auto ni) {
          static_for<4>([&](auto gg) {
            const int lc = wn * (NI * 32) + ni * 32 + gg * 8 + fhalf * 4;
            ev[mi & 1][ni][gg] = *(const gu2*)(Et + int(blk_index(il, lc, lde32)));
          });
        });
      };
      if constexpr (PK == kProdSquare) load_e(std::integral_constant<int, 0>{});
      auto write_round = [&](auto mi_c, auto diag_c) {
        constexpr int mi = decltype(mi_c)::value;
        constexpr bool DIAG = decltype(diag_c)::value;
        const int il = wm * (MI * 32) + mi * 32 + frow;  // tile row of this lane
        if constexpr (PK == kProdSquare && mi + 1 < MI) load_e(std::integral_constant<int, mi + 1>{});
        static_for<NI>([&](auto ni_c) {
          constexpr int ni = decltype(ni_c)::value;
          static_for<4>([&](auto gg_c) {
            constexpr int gg = decltype(gg_c)::value;
            float v0 = alpha * acc[mi][ni][4 * gg + 0];
            float v1 = alpha * acc[mi][ni][4 * gg + 1];
            float v2 = alpha * acc[mi][ni][4 * gg + 2];
            float v3 = alpha * acc[mi][ni][4 * gg + 3];
            if constexpr (PK == kProdSquare) {
              const u32x2 e = ev[mi & 1][ni][gg];
              v0 += beta * __uint_as_float(e.x << 16);
              v1 += beta * __uint_as_float(e.x & 0xffff0000u);
              v2 += beta * __uint_as_float(e.y << 16);
              v3 += beta * __uint_as_float(e.y & 0xffff0000u);
            }
            if constexpr (DIAG) {
              const int lc = wn * (NI * 32) + ni * 32 + gg * 8 + fhalf * 4;
              if (il == lc + 0) v0 += diag;
              if (il == lc + 1) v1 += diag;
              if (il == lc + 2) v2 += diag;
              if (il == lc + 3) v3 += diag;
            }
            // column block ni, chunk gg of this lane's slab row (chunk index swizzled)
            const int off = wr_base + ni * 1024 + (((gg ^ wr_sw) - wr_sw) << 4);
            *(l2x*)(slab + off) = u32x2{pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
          });
        });
      };
      static_for<MI>([&](auto mi_c) {
        constexpr int mi = decltype(mi_c)::value;
        if (PK == kProdSquare && diag != 0.0f)
          write_round(mi_c, std::true_type{});
        else
          write_round(mi_c, std::false_type{});
        MFSDP_WAIT_LGKM0();
        __builtin_amdgcn_s_barrier();
        if (Ct) {
#pragma unroll
          for (int bb = 0; bb < BPW; ++bb) {
            const int blk = w * BPW + bb, sp = blk / (TB / 32), cb = blk % (TB / 32);
            const u32x4 val = *(l4x*)(slab + (blk << 10) + rd_off);
            const int dr = (sp >> 1) * (MI * 32) + mi * 32 + (sp & 1) * 16 + row_in;
            *(gu4*)(Ct + int(blk_index(dr, cb * 32 + ch * 8, ldc32))) = val;
          }
        }
        if (Tt) {
#pragma unroll
          for (int bb = 0; bb < BPW; ++bb) {
            // transposed block tb: rows jp * 16 .. + 15 (tile columns), columns: the 32 tile rows
            // of wave row g2 in this round
            const int tb = w * BPW + bb, jp = tb >> 1, g2 = tb & 1;
            const int sr0 = g2 * 32 + tg * 8 + tr_r;
            const int cc = jp * 16 + tr_c * 4;
            const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lbf4*)(slab + slab_off(sr0, cc)));
            const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lbf4*)(slab + slab_off(sr0 + 4, cc)));
            const u32x4 val = __builtin_bit_cast(u32x4, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            *(gu4*)(Tt + int(blk_index(jp * 16 + til, g2 * (MI * 32) + mi * 32 + tg * 8, ldtd32))) = val;
          }
        }
        __builtin_amdgcn_s_barrier();  // slab reads done before the next round overwrites it
      });
      if (!has_next) break;
      cur = nxt;
      continue;
    }
    if constexpr (PK == kProdApply) {
      // Parameters the staged update does not take (fp32 parameters, or n % 8 != 0): straight from
      // the accumulators, 4 elements per lane and group; a tall parameter takes the quad-transposed
      // values. (Compile-time loops: every acc index must be a constant for acc to stay in registers.)
      static_for<MI>([&](auto mi_c) {
        constexpr int mi = decltype(mi_c)::value;
        const int64_t i = int64_t(bi) * TB + wm * (MI * 32) + mi * 32 + frow;
        const int64_t iq = i - q;  // first row of this lane quad
        static_for<NI>([&](auto ni_c) {
          constexpr int ni = decltype(ni_c)::value;
          static_for<4>([&](auto gg_c) {
            constexpr int gg = decltype(gg_c)::value;
            const int64_t j = int64_t(bj) * TB + wn * (NI * 32) + ni * 32 + gg * 8 + fhalf * 4;
            float v0 = alpha * acc[mi][ni][4 * gg + 0];
            float v1 = alpha * acc[mi][ni][4 * gg + 1];
            float v2 = alpha * acc[mi][ni][4 * gg + 2];
            float v3 = alpha * acc[mi][ni][4 * gg + 3];
            if (fa_t) {
              quad_transpose(v0, v1, v2, v3);
              apply4(*fa, j + q, iq, v0, v1, v2, v3);  // lane q: column j + q at rows iq .. iq + 3
            } else {
              apply4(*fa, i, j, v0, v1, v2, v3);
            }
          });
        });
      });
    }
    if (!has_next) break;
    cur = nxt;
  }
  // nothing of this workgroup may still be in flight when it exits
  MFSDP_WAIT_VMCNT(0);
}
#undef MFSDP_WAIT_VMCNT
#undef MFSDP_WAIT_LGKM0

// Second pass of a split Gram product (TB x TB tiles): one 256-thread workgroup per (job, 16-row
// slab of the tile). Thread t adds the nks partials of 4 consecutive columns 4 (t % (TB / 4)) of rows
// t / (TB / 4) + (1024 / TB) i in range order, scales as the Gram epilogue does and stores 8 bytes of
// bf16 into the tile; an off-diagonal tile's slab also goes through LDS to its mirror, where it is one
// 32-byte row piece per tile column (threads t < TB).
constexpr int kSumSlab = 16;
template <int TB>
__global__ __launch_bounds__(256) void gram_sum_kernel(const GemmDesc* __restrict__ descs,
                                                       const TileRef* __restrict__ jobs, int parity,
                                                       int first) {
  typedef float f32x4s __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) const f32x4s gcf4s;
  constexpr int TPR = TB / 4;          // threads per row
  constexpr int RPP = 256 / TPR;       // rows per pass
  __shared__ float tt[kSumSlab][TB + 1];
  const TileRef job = jobs[blockIdx.x / (TB / kSumSlab)];
  const int slab = blockIdx.x % (TB / kSumSlab);
  const GemmDesc& dd = descs[job.e];
  const int bi = job.bi, bj = job.bj, nks = dd.nks;
  const float alpha = dd.alpha * (first ? scale_pow(dd.scale, dd.alpha_scale_pow) : 1.0f);
  const float* part = dd.part + int64_t(upper_index(bi, bj, dd.tiles_m)) * nks * (TB * TB);
  gu16* C = (gu16*)dd.C[parity];
  const int64_t ldc = dd.ldc;
  const int t = threadIdx.x, c4 = (t % TPR) * 4;
#pragma unroll
  for (int i = 0; i < kSumSlab / RPP; ++i) {
    const int rl = t / TPR + RPP * i, r = slab * kSumSlab + rl;
    f32x4s a = *(gcf4s*)(part + r * TB + c4);
    for (int ks = 1; ks < nks; ++ks) a += *(gcf4s*)(part + int64_t(ks) * (TB * TB) + r * TB + c4);
    a *= alpha;
    *(gu2*)(C + blk_index(int64_t(bi) * TB + r, int64_t(bj) * TB + c4, ldc)) =
        u32x2{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3])};
    tt[rl][c4] = a[0];
    tt[rl][c4 + 1] = a[1];
    tt[rl][c4 + 2] = a[2];
    tt[rl][c4 + 3] = a[3];
  }
  if (bi == bj) return;  // (uniform) the diagonal tile is whole
  __syncthreads();
  if (t >= TB) return;
  // mirror row bj * TB + t, columns bi * TB + kSumSlab slab .. + kSumSlab - 1: part of one row of a
  // 16 x 32 block
  uint32_t w[kSumSlab / 2];
#pragma unroll
  for (int k = 0; k < kSumSlab / 2; ++k) w[k] = pack_bf16x2(tt[2 * k][t], tt[2 * k + 1][t]);
  gu4* dst = (gu4*)(C + blk_index(int64_t(bj) * TB + t, int64_t(bi) * TB + slab * kSumSlab, ldc));
#pragma unroll
  for (int k = 0; k < kSumSlab / 8; ++k) dst[k] = u32x4{w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]};
}

// fp32 NS products on fp32 MFMA. One 64 x 64 output tile per 256-thread workgroup: 4 waves of
// 32 x 32 (v_mfma_f32_32x32x2f32), K steps of 32 double-buffered in LDS with the next step's 16-byte
// global loads held in registers. The K index inside a step is permuted identically on both
// operands (lane half h of MFMA q in group g takes k = 8 g + 4 h + q), so each lane reads its
// fragments as 16-byte vectors; rows' eight 16-byte chunks are XOR-permuted by
// (r & 7) ^ ((r >> 3) & 1) in LDS (conflict-free for 32 and 64 banks). The epilogue follows the
// problem description: C = alpha P Q^T + beta E (+ the square's diagonal term), upper tiles of
// symmetric products with mirrored stores, the transposed output CT; transposed stores go through
// an LDS tile so that they are row-contiguous.
__device__ __forceinline__ int f32_slot(int r, int chunk) {
  return r * 8 + (chunk ^ ((r & 7) ^ ((r >> 3) & 1)));
}

__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmDesc* __restrict__ descs, int count,
                                                       int parity, int first, int last, float ca,
                                                       float cb, float cc) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  typedef float f32x16 __attribute__((ext_vector_type(16)));
  typedef __attribute__((address_space(1))) float gf32;
  typedef __attribute__((address_space(1))) const f32x4 gcf4;
  __shared__ f32x4 lds[2][2][64 * 8];  // [stage][P, Q][slot]: 32 KiB
  __shared__ float tt[64][65];          // transposition tile
  const int e = find_entry(descs, count, blockIdx.x);
  const GemmDesc& dd = descs[e];
  const int lt = blockIdx.x - dd.tile_begin;
  int bi, bj;
  tile_coords(dd, lt, bi, bj);
  const gf32* P = (const gf32*)dd.P[parity];
  const gf32* Q = (const gf32*)dd.Q[parity];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int fr = lane & 31, fh = lane >> 5;
  // global loads of one K step: the 64 x 32 slice of a panel-blocked operand is four 16 x 32 blocks
  // (2 KiB each); float4 f = t + 256 j covers block f >> 7, row (f >> 3) & 15, chunk f & 7
  const int64_t prow0 = int64_t(bi) * 64, qrow0 = int64_t(bj) * 64;
  f32x4 ra[2], rb[2];
  auto gload = [&](int k0) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int f = t + 256 * j;
      const int r = (f >> 7) * 16 + ((f >> 3) & 15), c = f & 7;
      ra[j] = *(gcf4*)(P + blk_index(prow0 + r, k0 + 4 * c, dd.ldp));
      rb[j] = *(gcf4*)(Q + blk_index(qrow0 + r, k0 + 4 * c, dd.ldq));
    }
  };
  auto lstore = [&](int s) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int f = t + 256 * j;
      const int slot = f32_slot((f >> 7) * 16 + ((f >> 3) & 15), f & 7);
      lds[s][0][slot] = ra[j];
      lds[s][1][slot] = rb[j];
    }
  };
  f32x16 acc = f32x16{};
  const int nk = dd.K / 32;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int s = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * 32);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 a = lds[s][0][f32_slot(wr * 32 + fr, 2 * g + fh)];
      const f32x4 b = lds[s][1][f32_slot(wc * 32 + fr, 2 * g + fh)];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[q], b[q], acc, 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(s ^ 1);
    __syncthreads();
  }
  // the square product (the only one with an addend) takes this step's coefficients
  const bool square = dd.E[parity] != nullptr;
  const float alpha = square ? cc : dd.alpha * (first ? scale_pow(dd.scale, dd.alpha_scale_pow) : 1.0f);
  const float beta = square ? cb : dd.beta * (first ? scale_pow(dd.scale, dd.beta_scale_pow) : 1.0f);
  const float diag = (square && dd.sym && bi == bj) ? ca : 0.0f;
  const gf32* E = (const gf32*)dd.E[parity];
  gf32* C = (gf32*)dd.C[parity];
  gf32* CT = (gf32*)dd.CT[parity];
  if (last) {
    if (!dd.last_c) C = nullptr;
    if (!dd.last_ct) CT = nullptr;
  }
  const bool mirror = dd.sym && bi != bj && C;
  // accumulator element v is tile row wr*32 + 8 (v / 4) + 4 h + v % 4, column wc*32 + lane % 32
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int i = wr * 32 + 8 * (v >> 2) + 4 * fh + (v & 3);
    const int j = wc * 32 + fr;
    const int64_t gi = prow0 + i, gj = qrow0 + j;
    float x = alpha * acc[v];
    if (E) x += beta * E[blk_index(gi, gj, dd.lde)];
    if (gi == gj) x += diag;
    if (C) C[blk_index(gi, gj, dd.ldc)] = x;
    tt[i][j] = x;
  }
  if (mirror || CT) {
    __syncthreads();
    // transposed tile: row qrow0 + j, columns prow0 + i (i across lanes)
    const int i = t & 63;
#pragma unroll 4
    for (int it = 0; it < 16; ++it) {
      const int j = (t >> 6) + 4 * it;
      const float x = tt[i][j];
      if (mirror) C[blk_index(qrow0 + j, prow0 + i, dd.ldc)] = x;
      if (CT) CT[blk_index(qrow0 + j, prow0 + i, dd.ldct)] = x;
    }
  }
}

}  // namespace

template <int NW, int TB, int PK>
void launch_bf16(const GemmDesc* d_descs, const TileRef* d_sched, int ngroups, int parity, int first_step,
                 int last_step, float ca, float cb, float cc, hipStream_t st) {
  hipLaunchKernelGGL((gemm_bf16_kernel<NW, TB, PK>), dim3(kGemmXcds * WaveGrid<NW, TB>::SLOTS),
                     dim3(NW * 64), 0, st, d_descs, d_sched, ngroups, parity, first_step, last_step, ca,
                     cb, cc);
}

hipError_t launch_gemm(const GemmDesc* d_descs, int count, int total_tiles, const TileRef* d_sched,
                       int ngroups, int ns_dtype, int product, int parity, int first_step,
                       int last_step, float ca, float cb, float cc, int tile, hipStream_t st) {
  if (total_tiles <= 0) return hipSuccess;
  if (ns_dtype == kDtBF16) {
    constexpr int W = kGemmWaves;
    constexpr int WS = kGemmWavesSmall, TS = kTileBF16Small;
    if (tile == TS) {
      if (product == kProdGram)
        launch_bf16<WS, TS, kProdGram>(d_descs, d_sched, ngroups, parity, first_step, last_step, ca, cb, cc, st);
      else if (product == kProdSquare)
        launch_bf16<WS, TS, kProdSquare>(d_descs, d_sched, ngroups, parity, first_step, last_step, ca, cb, cc, st);
      else
        return hipErrorInvalidValue;
    } else if (product == kProdGram)
      launch_bf16<W, BT, kProdGram>(d_descs, d_sched, ngroups, parity, first_step, last_step, ca, cb, cc, st);
    else if (product == kProdSquare)
      launch_bf16<W, BT, kProdSquare>(d_descs, d_sched, ngroups, parity, first_step, last_step, ca, cb, cc, st);
    else if (product == kProdUpdate)
      launch_bf16<W, BT, kProdUpdate>(d_descs, d_sched, ngroups, parity, first_step, last_step, ca, cb, cc, st);
    else
      launch_bf16<W, BT, kProdApply>(d_descs, d_sched, ngroups, parity, first_step, last_step, ca, cb, cc, st);
  } else
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(total_tiles), dim3(256), 0, st, d_descs, count,
                       parity, first_step, last_step, ca, cb, cc);
  return hipGetLastError();
}

hipError_t launch_gram_sum(const GemmDesc* d_descs, const TileRef* d_jobs, int njobs, int parity,
                           int first, int tile, hipStream_t st) {
  if (njobs <= 0) return hipSuccess;
  if (tile == kTileBF16Small)
    hipLaunchKernelGGL(gram_sum_kernel<kTileBF16Small>, dim3(njobs * (kTileBF16Small / kSumSlab)), dim3(256),
                       0, st, d_descs, d_jobs, parity, first);
  else
    hipLaunchKernelGGL(gram_sum_kernel<BT>, dim3(njobs * (BT / kSumSlab)), dim3(256), 0, st, d_descs,
                       d_jobs, parity, first);
  return hipGetLastError();
}

}  // namespace mfsdp
