// Host side of the C ABI declared in include/mfsdp.h: argument validation (all before any
// launch), workspace planning, descriptor upload and the launch sequence of the owner step.
//
// Launch sequence of mfsdp_muon_step (all on the caller's stream):
//   1. descriptor upload (pinned staging slot -> workspace)
//   2. prep     : momentum EMA + Nesterov, Sum u^2 partials, u in both layouts   (one launch)
//   3. norm     : per-matrix scale 1 / max(||u||_F, eps)                          (one launch)
//   4. K times  : Gram A = X X^T, square B = bA + cAA, update X' = aX + BX        (3 launches
//                 per step, each grouped over every matrix, heaviest tiles first)
//   5. apply    : p <- p (1 - lr wd) - lr f O                                     (one launch)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/mfsdp.h"
#include "mfsdp_internal.h"

using namespace mfsdp;

static_assert(MFSDP_MAX_GRAD_PARTS == kMaxGradParts, "gradient part limit of the ABI and the descriptor");

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

}  // namespace

namespace mfsdp {
int set_last_error(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}
}  // namespace mfsdp

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x, size_t a = kAlign) { return (x + a - 1) / a * a; }
inline int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

bool valid_dtype(int32_t dt) { return dt == MFSDP_F32 || dt == MFSDP_BF16; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------------------------------------
// Workspace plan for one NS problem (shared by the Muon step and standalone NS).
struct NsPlan {
  int64_t m, n, r, s, r_pad, s_pad;
  bool tall;
  int es;                   // element size of the NS dtype
  size_t off_x[2], off_xt[2], off_g, off_h, off_partials, off_scale;
  int prep_tiles_m, prep_tiles_n;
  size_t bytes;             // total for this problem
};

NsPlan plan_ns(int64_t m, int64_t n, int ns_dtype, size_t base) {
  NsPlan p{};
  p.m = m;
  p.n = n;
  p.tall = m > n;
  p.r = std::min(m, n);
  p.s = std::max(m, n);
  const int tile = ns_dtype == MFSDP_BF16 ? kTileBF16 : kTileF32;
  p.r_pad = round_up(p.r, tile);
  p.s_pad = round_up(p.s, tile);
  p.es = ns_dtype == MFSDP_BF16 ? 2 : 4;
  const size_t xb = align_up(size_t(p.r_pad) * size_t(p.s_pad) * p.es);
  const size_t gb = align_up(size_t(p.r_pad) * size_t(p.r_pad) * p.es);
  const int64_t rows = p.tall ? p.s_pad : p.r_pad, cols = p.tall ? p.r_pad : p.s_pad;
  p.prep_tiles_m = int(rows / kPrepRows);
  p.prep_tiles_n = int(cols / (ns_dtype == MFSDP_BF16 ? kPrepColsBF16 : kPrepColsF32));
  size_t o = base;
  p.off_x[0] = o; o += xb;
  p.off_x[1] = o; o += xb;
  p.off_xt[0] = o; o += xb;
  p.off_xt[1] = o; o += xb;
  p.off_g = o; o += gb;
  p.off_h = o; o += gb;
  p.off_partials = o; o += align_up(size_t(p.prep_tiles_m) * p.prep_tiles_n * sizeof(float));
  p.off_scale = o; o += kAlign;
  p.bytes = o - base;
  return p;
}

// Descriptor region at the start of the workspace.
struct DescLayout {
  size_t off_prep, off_norm, off_gemm[3], off_apply, off_sched[3], off_jobs, bytes;
  int ngroups[3];
  int njobs;  // tiles of the split Gram problems (second pass)
};


DescLayout plan_descs(int64_t count, const size_t sched_bytes[3], int njobs) {
  DescLayout d{};
  size_t o = 0;
  d.off_prep = o; o += align_up(sizeof(PrepDesc) * count);
  d.off_norm = o; o += align_up(sizeof(NormDesc) * count);
  for (int k = 0; k < 3; ++k) { d.off_gemm[k] = o; o += align_up(sizeof(GemmDesc) * count); }
  d.off_apply = o; o += align_up(sizeof(ApplyDesc) * count);
  for (int k = 0; k < 3; ++k) { d.off_sched[k] = o; o += align_up(sched_bytes[k]); }
  d.off_jobs = o; o += align_up(sizeof(TileRef) * size_t(njobs));
  d.njobs = njobs;
  d.bytes = o;
  return d;
}

// ---------------------------------------------------------------------------------------------
// Pinned staging ring for descriptor uploads. A slot is reused only after the copy that read it
// has completed (event per slot).
class StagingRing {
 public:
  static constexpr int kSlots = 16;
  int acquire(size_t bytes, void** host, hipStream_t st) {
    (void)st;
    std::lock_guard<std::mutex> lk(mu_);
    const int s = next_;
    next_ = (next_ + 1) % kSlots;
    Slot& sl = slots_[s];
    if (sl.event) {
      hipError_t e = hipEventSynchronize(sl.event);
      if (e != hipSuccess) return fail(MFSDP_E_HIP, "staging event: %s", hipGetErrorString(e));
    }
    if (sl.cap < bytes) {
      if (sl.ptr) (void)hipHostFree(sl.ptr);
      sl.ptr = nullptr;
      sl.cap = 0;
      size_t cap = std::max<size_t>(bytes, 64 * 1024);
      hipError_t e = hipHostMalloc(&sl.ptr, cap, hipHostMallocDefault);
      if (e != hipSuccess) return fail(MFSDP_E_HIP, "hipHostMalloc: %s", hipGetErrorString(e));
      sl.cap = cap;
    }
    if (!sl.event) {
      hipError_t e = hipEventCreateWithFlags(&sl.event, hipEventDisableTiming);
      if (e != hipSuccess) return fail(MFSDP_E_HIP, "hipEventCreate: %s", hipGetErrorString(e));
    }
    *host = sl.ptr;
    return s;
  }
  int upload(int slot, void* dst, size_t bytes, hipStream_t st) {
    Slot& sl = slots_[slot];
    hipError_t e = hipMemcpyAsync(dst, sl.ptr, bytes, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return fail(MFSDP_E_HIP, "descriptor upload: %s", hipGetErrorString(e));
    e = hipEventRecord(sl.event, st);
    if (e != hipSuccess) return fail(MFSDP_E_HIP, "hipEventRecord: %s", hipGetErrorString(e));
    return MFSDP_OK;
  }

 private:
  struct Slot {
    void* ptr = nullptr;
    size_t cap = 0;
    hipEvent_t event = nullptr;
  };
  std::mutex mu_;
  int next_ = 0;
  Slot slots_[kSlots];
};

StagingRing& ring() {
  static StagingRing* r = new StagingRing();  // lives until process exit
  return *r;
}

int check_hp(const mfsdp_muon_hparams* hp) {
  if (!hp) return fail(MFSDP_E_INVALID, "hparams is NULL");
  if (!(hp->lr >= 0.0) || !std::isfinite(hp->lr)) return fail(MFSDP_E_INVALID, "lr must be >= 0");
  if (!(hp->weight_decay >= 0.0) || !std::isfinite(hp->weight_decay))
    return fail(MFSDP_E_INVALID, "weight_decay must be >= 0");
  if (!(hp->momentum >= 0.0 && hp->momentum < 1.0))
    return fail(MFSDP_E_INVALID, "momentum must be in [0, 1)");
  if (hp->nesterov != 0 && hp->nesterov != 1) return fail(MFSDP_E_INVALID, "nesterov must be 0 or 1");
  if (hp->ns_steps < 0 || hp->ns_steps >= 100) return fail(MFSDP_E_INVALID, "ns_steps must be in [0, 100)");
  if (hp->ns_schedule) {
    for (int i = 0; i < 3 * hp->ns_steps; ++i)
      if (!std::isfinite(hp->ns_schedule[i]))
        return fail(MFSDP_E_INVALID, "ns_schedule entry %d is not finite", i);
  } else if (!std::isfinite(hp->a) || !std::isfinite(hp->b) || !std::isfinite(hp->c)) {
    return fail(MFSDP_E_INVALID, "NS coefficients must be finite");
  }
  if (!(hp->eps > 0.0) || !std::isfinite(hp->eps)) return fail(MFSDP_E_INVALID, "eps must be > 0");
  if (hp->lr_adjust < MFSDP_LR_NONE || hp->lr_adjust > MFSDP_LR_MATCH_RMS_ADAMW)
    return fail(MFSDP_E_INVALID, "unknown lr_adjust %d", hp->lr_adjust);
  if (!valid_dtype(hp->ns_dtype)) return fail(MFSDP_E_INVALID, "unknown ns_dtype %d", hp->ns_dtype);
  return MFSDP_OK;
}

constexpr int64_t kMaxDim = int64_t(1) << 20;   // per-side limit (index math stays in int32 tiles)

int check_shape(int64_t m, int64_t n, const char* what, int64_t i) {
  if (m <= 0 || n <= 0) return fail(MFSDP_E_INVALID, "%s %lld: shape %lldx%lld must be positive", what,
                                    (long long)i, (long long)m, (long long)n);
  if (m > kMaxDim || n > kMaxDim)
    return fail(MFSDP_E_INVALID, "%s %lld: side larger than %lld", what, (long long)i, (long long)kMaxDim);
  return MFSDP_OK;
}

// need_grad: the entries' grad pointers are read (0 for the workspace query and the fused
// reduction, which read no entry grad)
int check_entries(const mfsdp_muon_entry* entries, int64_t count, bool need_grad = true) {
  if (count < 0) return fail(MFSDP_E_INVALID, "count must be >= 0");
  if (count > 0 && !entries) return fail(MFSDP_E_INVALID, "entries is NULL");
  if (count > (1 << 20)) return fail(MFSDP_E_INVALID, "too many entries");
  int64_t units = 0;  // bound on the 64 x 64 tiles of any one grouped launch (grid and int32 counters)
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_muon_entry& e = entries[i];
    if (!e.param || (need_grad && !e.grad) || !e.momentum)
      return fail(MFSDP_E_INVALID, "entry %lld: NULL pointer", (long long)i);
    int st = check_shape(e.m, e.n, "entry", i);
    if (st) return st;
    units += (round_up(e.m, kTileBF16) / 64) * (round_up(e.n, kTileBF16) / 64);
    if (units > (int64_t(1) << 30))
      return fail(MFSDP_E_INVALID, "the entries of one call exceed 2^30 tiles per launch");
    if (!valid_dtype(e.param_dtype) || !valid_dtype(e.grad_dtype))
      return fail(MFSDP_E_INVALID, "entry %lld: unsupported dtype", (long long)i);
    if (!aligned16(e.param) || (need_grad && !aligned16(e.grad)) || !aligned16(e.momentum) ||
        (e.update_out && !aligned16(e.update_out)))
      return fail(MFSDP_E_INVALID, "entry %lld: pointers must be 16-byte aligned", (long long)i);
  }
  return MFSDP_OK;
}

double lr_factor(int64_t m, int64_t n, int mode) {
  if (mode == MFSDP_LR_ORIGINAL) return std::sqrt(std::max(1.0, double(m) / double(n)));
  if (mode == MFSDP_LR_MATCH_RMS_ADAMW) return 0.2 * std::sqrt(double(std::max(m, n)));
  return 1.0;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(MFSDP_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Builds and enqueues the NS pipeline for a set of problems that already have their prep
// descriptors filled. Shared by the Muon step and standalone NS.
// Problem order of one NS product: heaviest K first (all tiles have the same size, so the work
// of a tile is proportional to K).
std::vector<int> phase_order(const std::vector<NsPlan>& plans, int phase) {
  std::vector<int> ord(plans.size());
  for (size_t i = 0; i < ord.size(); ++i) ord[i] = int(i);
  std::stable_sort(ord.begin(), ord.end(), [&](int x, int y) {
    const int64_t kx = phase == 0 ? plans[x].s_pad : plans[x].r_pad;
    const int64_t ky = phase == 0 ? plans[y].s_pad : plans[y].r_pad;
    return kx > ky;
  });
  return ord;
}

// Everything about a call that follows from the shapes and the NS dtype: per-matrix buffers,
// the problem order and tile schedule of each NS product, and the descriptor region layout.
struct Plan {
  std::vector<NsPlan> ns;
  std::vector<int> order[3];
  std::vector<TileRef> sched[3];
  int tiles[3] = {0, 0, 0};
  int tile[3] = {0, 0, 0};     // output tile of each product's launch
  std::vector<int> split;      // per Gram problem (launch order): K ranges per tile
  std::vector<size_t> part;    // per Gram problem: offset of its partial tiles (split ones)
  std::vector<TileRef> jobs;   // the split problems' upper tiles (second pass)
  DescLayout dl{};
  size_t bytes = 0;
};

// On the bf16 path a Gram launch with fewer tiles than the persistent grid has workgroups may split
// long contractions (gram_splits); the split problems' partial tiles follow the per-matrix buffers
// and take at most a quarter of their bytes. When the r x r products' 128 x 128 tiles fit one round
// of the two-workgroups-per-CU grid, the Gram and square launches run on those (small shares: four
// times the tiles of launches that would leave most CUs idle, each with a quarter of the epilogue).
template <typename ShapeAt>
Plan make_plan(int64_t count, int ns_dtype, ShapeAt shape_at) {
  Plan P;
  std::vector<NsPlan> shapes;
  for (int64_t i = 0; i < count; ++i) {
    int64_t m, n;
    shape_at(i, m, n);
    shapes.push_back(plan_ns(m, n, ns_dtype, 0));
  }
  const bool bf = ns_dtype == MFSDP_BF16;
  int64_t small_tiles = 0;  // upper 128 x 128 tiles of the r x r products
  for (const NsPlan& p : shapes) {
    const int64_t t = p.r_pad / kTileBF16Small;
    small_tiles += t * (t + 1) / 2;
  }
  const int64_t small_slots = int64_t(kGemmXcds) * 2 * kGemmSlots;
  size_t sched_bytes[3] = {0, 0, 0};
  for (int ph = 0; ph < 3; ++ph) {
    const bool small = bf && ph < 2 && small_tiles <= small_slots;
    const int tile = !bf ? kTileF32 : small ? kTileBF16Small : kTileBF16;
    P.tile[ph] = tile;
    P.order[ph] = phase_order(shapes, ph);
    std::vector<TileGrid> grids;
    std::vector<int> pos;
    std::vector<int64_t> cost;
    for (int k = 0; k < int(count); ++k) {
      const NsPlan& p = shapes[P.order[ph][k]];
      const int tr = int(p.r_pad / tile), ts = int(p.s_pad / tile);
      const TileGrid g = ph == 2 ? TileGrid{tr, ts, false} : TileGrid{tr, tr, true};
      grids.push_back(g);
      pos.push_back(k);
      cost.push_back(ph == 0 ? p.s_pad : p.r_pad);
      P.tiles[ph] += g.sym ? g.tm * (g.tm + 1) / 2 : g.tm * g.tn;
    }
    if (ph == 0) {
      P.split.assign(size_t(count), 1);
      if (ns_dtype == MFSDP_BF16) {
        std::vector<int64_t> tl, kl;
        for (const TileGrid& g : grids) tl.push_back(int64_t(g.tm) * (g.tm + 1) / 2);
        for (int64_t c : cost) kl.push_back(c);
        size_t base = 0;
        for (const NsPlan& q : shapes) base += q.bytes;
        const size_t part_bytes = size_t(tile) * tile * sizeof(float);
        P.split = gram_splits(tl, kl, int64_t(base / 4 / part_bytes),
                              small ? small_slots : int64_t(kGemmXcds) * kGemmSlots);
      }
      for (int k = 0; k < int(count); ++k)
        if (P.split[size_t(k)] > 1)
          for (int bi = 0; bi < grids[size_t(k)].tm; ++bi)
            for (int bj = bi; bj < grids[size_t(k)].tm; ++bj)
              P.jobs.push_back(TileRef{k, int16_t(bi), int16_t(bj), 0, 0});
    }
    if (bf && small) {
      // at most one tile per CU when they fit: groups of kGemmSlots tiles on the 2 x kGemmSlots slots
      int64_t n = 0;
      for (size_t k = 0; k < grids.size(); ++k)
        n += int64_t(grids[k].tm) * (grids[k].tm + 1) / 2 * (ph == 0 ? P.split[k] : 1);
      const int fill = n <= int64_t(kGemmXcds) * kGemmSlots ? kGemmSlots : 2 * kGemmSlots;
      P.sched[ph] = build_schedule(pos, grids, cost, ph == 0 ? &P.split : nullptr, 2 * kGemmSlots,
                                   2 * kGroupRows, fill);
    } else if (bf)
      P.sched[ph] = build_schedule(pos, grids, cost, ph == 0 ? &P.split : nullptr);
    sched_bytes[ph] = P.sched[ph].size() * sizeof(TileRef);
  }
  P.dl = plan_descs(count, sched_bytes, int(P.jobs.size()));
  for (int ph = 0; ph < 3; ++ph)
    P.dl.ngroups[ph] = int(P.sched[ph].size() / (P.tile[ph] == kTileBF16Small ? 2 * kGemmSlots : kGemmSlots));
  size_t o = P.dl.bytes;
  for (int64_t i = 0; i < count; ++i) {
    P.ns.push_back(plan_ns(shapes[i].m, shapes[i].n, ns_dtype, o));
    o += P.ns.back().bytes;
  }
  P.part.assign(size_t(count), 0);
  for (int k = 0; k < int(count); ++k) {
    const int f = P.split[size_t(k)];
    if (f <= 1) continue;
    const int64_t tr = shapes[size_t(P.order[0][size_t(k)])].r_pad / P.tile[0];
    P.part[size_t(k)] = o;
    o += align_up(size_t(tr * (tr + 1) / 2) * size_t(f) * P.tile[0] * P.tile[0] * sizeof(float));
  }
  P.bytes = o;
  return P;
}

// Coefficients of every NS step: the schedule if given, else the fixed triple.
std::vector<double> step_coeffs(double a, double b, double c, int steps, const double* schedule) {
  std::vector<double> v(3 * size_t(steps));
  for (int k = 0; k < steps; ++k) {
    v[3 * k] = schedule ? schedule[3 * k] : a;
    v[3 * k + 1] = schedule ? schedule[3 * k + 1] : b;
    v[3 * k + 2] = schedule ? schedule[3 * k + 2] : c;
  }
  return v;
}

// On the bf16 path with at least one NS step the last update product applies the parameter update
// in its epilogue (from the fp32 accumulators); otherwise a separate apply pass reads the iterate.
bool apply_fused(int ns_dtype, int steps) { return ns_dtype == MFSDP_BF16 && steps >= 1; }

// Descriptors of the three products, stored in the phase's problem order; the schedules refer
// to problems by that position.
void fill_gemm_descs(const Plan& P, uint8_t* ws, const mfsdp_muon_hparams& hp, uint8_t* h) {
  const int n = int(P.ns.size());
  for (int phase = 0; phase < 3; ++phase) {
    const int tile = P.tile[phase];
    GemmDesc* out = reinterpret_cast<GemmDesc*>(h + P.dl.off_gemm[phase]);
    const std::vector<int>& ord = P.order[phase];
    int begin = 0;
    for (int k = 0; k < n; ++k) {
      const NsPlan& p = P.ns[ord[k]];
      GemmDesc d{};
      const int tr = int(p.r_pad / tile), ts = int(p.s_pad / tile);
      for (int par = 0; par < 2; ++par) {
        uint8_t* xin = ws + p.off_x[par];
        uint8_t* xtin = ws + p.off_xt[par];
        uint8_t* xout = ws + p.off_x[par ^ 1];
        uint8_t* xtout = ws + p.off_xt[par ^ 1];
        if (phase == 0) {         // A = X X^T
          d.P[par] = xin; d.Q[par] = xin; d.E[par] = nullptr;
          d.C[par] = ws + p.off_g; d.CT[par] = nullptr;
        } else if (phase == 1) {  // B' = c A A + b A + a I
          d.P[par] = ws + p.off_g; d.Q[par] = ws + p.off_g; d.E[par] = ws + p.off_g;
          d.C[par] = ws + p.off_h; d.CT[par] = nullptr;
        } else {                  // X' = B' X (= a X + B X), stored as X' and X'^T
          d.P[par] = ws + p.off_h; d.Q[par] = xtin; d.E[par] = nullptr;
          d.C[par] = xout; d.CT[par] = xtout;
        }
      }
      d.scale = reinterpret_cast<const float*>(ws + p.off_scale);
      if (phase == 0) {
        d.ldp = d.ldq = p.s_pad; d.lde = 0; d.ldc = p.r_pad; d.ldct = 0;
        d.M = d.N = int(p.r_pad); d.K = int(p.s_pad);
        d.alpha = 1.0f; d.beta = 0.0f; d.alpha_scale_pow = 2; d.beta_scale_pow = 0;
        d.sym = 1; d.tiles_m = d.tiles_n = tr;
        d.tile_count = tr * (tr + 1) / 2;
        d.last_c = 1; d.last_ct = 0;
        d.nks = P.split[size_t(k)];
        d.part = d.nks > 1 ? reinterpret_cast<float*>(ws + P.part[size_t(k)]) : nullptr;
      } else if (phase == 1) {
        d.ldp = d.ldq = d.lde = d.ldc = p.r_pad; d.ldct = 0;
        d.M = d.N = d.K = int(p.r_pad);
        d.alpha = 0.0f; d.beta = 0.0f;  // the step's (a, b, c) come with each launch
        d.alpha_scale_pow = 0; d.beta_scale_pow = 0;
        d.sym = 1; d.tiles_m = d.tiles_n = tr;
        d.tile_count = tr * (tr + 1) / 2;
        d.last_c = 1; d.last_ct = 0;
      } else {
        d.ldp = p.r_pad; d.ldq = p.r_pad; d.lde = 0; d.ldc = p.s_pad; d.ldct = p.r_pad;
        d.M = int(p.r_pad); d.N = int(p.s_pad); d.K = int(p.r_pad);
        d.alpha = 1.0f; d.beta = 0.0f; d.alpha_scale_pow = 1; d.beta_scale_pow = 0;
        d.sym = 0; d.tiles_m = tr; d.tiles_n = ts;
        d.tile_count = tr * ts;
        // the final iterate is read in the parameter's orientation only
        d.last_c = p.tall ? 0 : 1;
        d.last_ct = p.tall ? 1 : 0;
        if (apply_fused(hp.ns_dtype, hp.ns_steps))
          d.fused = reinterpret_cast<const ApplyDesc*>(ws + P.dl.off_apply) + ord[k];
      }
      d.tile_begin = begin;
      begin += d.tile_count;
      out[k] = d;
    }
    if (!P.sched[phase].empty())
      std::memcpy(h + P.dl.off_sched[phase], P.sched[phase].data(),
                  P.sched[phase].size() * sizeof(TileRef));
  }
  if (!P.jobs.empty()) std::memcpy(h + P.dl.off_jobs, P.jobs.data(), P.jobs.size() * sizeof(TileRef));
}

PrepDesc make_prep(const NsPlan& p, uint8_t* ws, const void* grad, int grad_dtype, float* momentum,
                   int tile_begin) {
  PrepDesc d{};
  d.grad = grad;
  d.momentum = momentum;
  // u in its stored orientation is X (wide) or X^T (tall); its transpose goes to the other one
  if (p.tall) {
    d.d_out = ws + p.off_xt[0]; d.ld_d = p.r_pad;
    d.t_out = ws + p.off_x[0];  d.ld_t = p.s_pad;
  } else {
    d.d_out = ws + p.off_x[0];  d.ld_d = p.s_pad;
    d.t_out = ws + p.off_xt[0]; d.ld_t = p.r_pad;
  }
  d.partials = reinterpret_cast<float*>(ws + p.off_partials);
  d.m = p.m;
  d.n = p.n;
  d.tiles_m = p.prep_tiles_m;
  d.tiles_n = p.prep_tiles_n;
  d.grad_dtype = grad_dtype;
  d.tile_begin = tile_begin;
  return d;
}

ApplyDesc make_apply(const NsPlan& p, uint8_t* ws, int steps, void* param, int param_dtype,
                     float* update_out, int mode, float decay, float step, int tile_begin) {
  ApplyDesc d{};
  const int par = steps & 1;  // parity of the buffer holding the final iterate
  if (p.tall) { d.o = ws + p.off_xt[par]; d.ld_o = p.r_pad; }
  else        { d.o = ws + p.off_x[par];  d.ld_o = p.s_pad; }
  d.param = param;
  d.update_out = update_out;
  d.scale = reinterpret_cast<const float*>(ws + p.off_scale);
  d.use_scale = steps == 0 ? 1 : 0;
  d.m = p.m;
  d.n = p.n;
  d.param_dtype = param_dtype;
  d.mode = mode;
  d.decay = decay;
  d.step = step;
  d.tiles_m = int((p.m + kApplyRows - 1) / kApplyRows);
  d.tiles_n = int((p.n + kApplyCols - 1) / kApplyCols);
  d.tile_begin = tile_begin;
  return d;
}

// Enqueue everything after the descriptors are in host staging memory `h`.
int record(void* const* events, int k, hipStream_t st) {
  if (!events || !events[k]) return MFSDP_OK;
  hipError_t e = hipEventRecord(static_cast<hipEvent_t>(events[k]), st);
  return e == hipSuccess ? MFSDP_OK : hip_fail(e, "hipEventRecord");
}

int upload_as_kernel_args(const uint8_t* host, size_t bytes, uint8_t* dst, hipStream_t st);

// coeffs: 3 * steps doubles, (a_k, b_k, c_k) of NS step k.
// Descriptors: slot >= 0 uploads them from that pinned staging slot; slot < 0 passes them from the
// host buffer `host_descs` as kernel arguments (the allocation-free step).
int enqueue_pipeline(const Plan& P, uint8_t* ws, int slot, int steps, const double* coeffs,
                     int ns_dtype, double beta, int nesterov, double eps, int prep_tiles,
                     int apply_tiles, hipStream_t st, void* const* events, bool reduce = false,
                     const uint8_t* host_descs = nullptr) {
  const int count = int(P.ns.size());
  const DescLayout& dl = P.dl;
  int rc = slot >= 0 ? ring().upload(slot, ws, dl.bytes, st) : upload_as_kernel_args(host_descs, dl.bytes, ws, st);
  if (rc) return rc;
  if ((rc = record(events, 0, st))) return rc;
  hipError_t e;
  e = launch_prep(reinterpret_cast<const PrepDesc*>(ws + dl.off_prep), count, prep_tiles, ns_dtype,
                  reduce ? 1 : 0, float(beta), float(1.0 - beta), nesterov, st);
  if (e != hipSuccess) return hip_fail(e, "prep launch");
  e = launch_norm(reinterpret_cast<const NormDesc*>(ws + dl.off_norm), count, float(eps), st);
  if (e != hipSuccess) return hip_fail(e, "norm launch");
  if ((rc = record(events, 1, st))) return rc;
  for (int k = 0; k < steps; ++k) {
    for (int ph = 0; ph < 3; ++ph) {
      // the last update of the bf16 path applies the parameter update in its epilogue (kind 3)
      const int kind = (ph == 2 && k == steps - 1 && apply_fused(ns_dtype, steps)) ? 3 : ph;
      e = launch_gemm(reinterpret_cast<const GemmDesc*>(ws + dl.off_gemm[ph]), count, P.tiles[ph],
                      reinterpret_cast<const TileRef*>(ws + dl.off_sched[ph]), dl.ngroups[ph],
                      ns_dtype, kind, k & 1, k == 0 ? 1 : 0, k == steps - 1 ? 1 : 0,
                      float(coeffs[3 * k]), float(coeffs[3 * k + 1]), float(coeffs[3 * k + 2]), P.tile[ph],
                      st);
      if (e != hipSuccess) return hip_fail(e, "NS GEMM launch");
      if (ph == 0 && dl.njobs > 0) {
        e = launch_gram_sum(reinterpret_cast<const GemmDesc*>(ws + dl.off_gemm[0]),
                            reinterpret_cast<const TileRef*>(ws + dl.off_jobs), dl.njobs, k & 1,
                            k == 0 ? 1 : 0, P.tile[0], st);
        if (e != hipSuccess) return hip_fail(e, "split Gram sum launch");
      }
    }
  }
  if ((rc = record(events, 2, st))) return rc;
  if (!apply_fused(ns_dtype, steps)) {
    e = launch_apply(reinterpret_cast<const ApplyDesc*>(ws + dl.off_apply), count, apply_tiles,
                     ns_dtype, st);
    if (e != hipSuccess) return hip_fail(e, "apply launch");
  }
  return record(events, 3, st);
}

int ns_impl(const void* x, int32_t x_dtype, void* out, int32_t out_dtype, int64_t m, int64_t n,
            const double* coeffs, int32_t steps, double eps, int32_t ns_dtype, void* workspace,
            size_t workspace_bytes, void* stream);

// The fused owner-side gradient reduction of mfsdp_muon_step_reduce (validated).
struct ReduceArgs {
  const void* const* parts;  // count * nparts device pointers
  int nparts;
  double scale;
  void* const* out;          // NULL or count pointers (each may be NULL)
};
int muon_impl(const mfsdp_muon_entry* entries, int64_t count, const mfsdp_muon_hparams* hp,
              void* workspace, size_t workspace_bytes, void* stream, void* const* events,
              const ReduceArgs* ra, bool in_scratch = false);

}  // namespace

extern "C" {

int mfsdp_abi_version(void) { return MFSDP_ABI_VERSION; }

#ifndef MFSDP_BUILD_ID
#define MFSDP_BUILD_ID "unknown"
#endif
const char* mfsdp_build_id(void) { return MFSDP_BUILD_ID; }

const char* mfsdp_last_error(void) { return g_last_error.c_str(); }

const char* mfsdp_status_string(int status) {
  switch (status) {
    case MFSDP_OK: return "MFSDP_OK";
    case MFSDP_E_INVALID: return "MFSDP_E_INVALID";
    case MFSDP_E_WORKSPACE: return "MFSDP_E_WORKSPACE";
    case MFSDP_E_HIP: return "MFSDP_E_HIP";
    default: return "MFSDP_E_UNKNOWN";
  }
}

size_t mfsdp_muon_workspace_size(const mfsdp_muon_entry* entries, int64_t count,
                                 const mfsdp_muon_hparams* hp) {
  g_last_error.clear();
  if (check_hp(hp) || check_entries(entries, count, false)) return 0;
  if (count == 0) return 0;
  return make_plan(count, hp->ns_dtype, [&](int64_t i, int64_t& m, int64_t& n) {
           m = entries[i].m;
           n = entries[i].n;
         }).bytes;
}

int mfsdp_muon_step(const mfsdp_muon_entry* entries, int64_t count, const mfsdp_muon_hparams* hp,
                    void* workspace, size_t workspace_bytes, void* stream) {
  return mfsdp_muon_step_timed(entries, count, hp, workspace, workspace_bytes, stream, nullptr);
}

int mfsdp_muon_step_timed(const mfsdp_muon_entry* entries, int64_t count,
                          const mfsdp_muon_hparams* hp, void* workspace, size_t workspace_bytes,
                          void* stream, void* const* events) {
  g_last_error.clear();
  return muon_impl(entries, count, hp, workspace, workspace_bytes, stream, events, nullptr);
}

int mfsdp_muon_step_reduce(const mfsdp_muon_entry* entries, int64_t count,
                           const void* const* grad_parts, int32_t nparts, double grad_scale,
                           void* const* reduced_out, const mfsdp_muon_hparams* hp, void* workspace,
                           size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (nparts < 1 || nparts > MFSDP_MAX_GRAD_PARTS)
    return fail(MFSDP_E_INVALID, "nparts must be in [1, %d]", MFSDP_MAX_GRAD_PARTS);
  if (!std::isfinite(grad_scale)) return fail(MFSDP_E_INVALID, "grad_scale must be finite");
  if (count > 0 && !grad_parts) return fail(MFSDP_E_INVALID, "grad_parts is NULL");
  for (int64_t i = 0; i < count; ++i) {
    for (int w = 0; w < nparts; ++w) {
      const void* pw = grad_parts[i * nparts + w];
      if (!pw || !aligned16(pw))
        return fail(MFSDP_E_INVALID, "entry %lld part %d: NULL or not 16-byte aligned", (long long)i, w);
    }
    if (reduced_out && reduced_out[i] && !aligned16(reduced_out[i]))
      return fail(MFSDP_E_INVALID, "entry %lld: reduced_out not 16-byte aligned", (long long)i);
  }
  const ReduceArgs ra{grad_parts, nparts, grad_scale, reduced_out};
  return muon_impl(entries, count, hp, workspace, workspace_bytes, stream, nullptr, &ra);
}

}  // extern "C"

namespace {

int scratch_address(void** out);

// in_scratch: the allocation-free step. The workspace is this device's static scratch array
// (`workspace` and `workspace_bytes` are ignored) and the descriptors travel as kernel arguments
// from ordinary host memory instead of through the pinned staging ring.
int muon_impl(const mfsdp_muon_entry* entries, int64_t count, const mfsdp_muon_hparams* hp,
              void* workspace, size_t workspace_bytes, void* stream, void* const* events,
              const ReduceArgs* ra, bool in_scratch) {
  int rc = check_hp(hp);
  if (rc) return rc;
  rc = check_entries(entries, count, ra == nullptr);
  if (rc) return rc;
  if (count == 0) return MFSDP_OK;
  const Plan P = make_plan(count, hp->ns_dtype, [&](int64_t i, int64_t& m, int64_t& n) {
    m = entries[i].m;
    n = entries[i].n;
  });
  const std::vector<NsPlan>& plans = P.ns;
  const size_t need = P.bytes;
  if (in_scratch) {
    if (need > size_t(MFSDP_NOALLOC_SCRATCH_BYTES))
      return fail(MFSDP_E_INVALID,
                  "these entries need %zu bytes of workspace; the allocation-free step holds at most "
                  "%zu (MFSDP_NOALLOC_SCRATCH_BYTES): use mfsdp_muon_step with a caller workspace",
                  need, size_t(MFSDP_NOALLOC_SCRATCH_BYTES));
    if ((rc = scratch_address(&workspace))) return rc;
    workspace_bytes = MFSDP_NOALLOC_SCRATCH_BYTES;
  }
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return fail(MFSDP_E_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
  if (workspace_bytes < need)
    return fail(MFSDP_E_WORKSPACE, "workspace too small: %zu < %zu bytes", workspace_bytes, need);

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const DescLayout& dl = P.dl;
  int slot = -1;
  std::vector<uint8_t> host_descs;
  uint8_t* h = nullptr;
  if (in_scratch) {
    host_descs.assign(dl.bytes, 0);
    h = host_descs.data();
  } else {
    void* hptr = nullptr;
    slot = ring().acquire(dl.bytes, &hptr, st);
    if (slot < 0) return slot;
    h = static_cast<uint8_t*>(hptr);
    std::memset(h, 0, dl.bytes);
  }

  auto* prep = reinterpret_cast<PrepDesc*>(h + dl.off_prep);
  auto* norm = reinterpret_cast<NormDesc*>(h + dl.off_norm);
  auto* apply = reinterpret_cast<ApplyDesc*>(h + dl.off_apply);
  int prep_tiles = 0, apply_tiles = 0;
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_muon_entry& en = entries[i];
    const NsPlan& p = plans[i];
    prep[i] = make_prep(p, ws, en.grad, en.grad_dtype, en.momentum, prep_tiles);
    if (ra) {
      prep[i].nparts = ra->nparts;
      prep[i].gscale = float(ra->scale);
      prep[i].gout = ra->out ? ra->out[i] : nullptr;
      for (int w = 0; w < ra->nparts; ++w) prep[i].parts[w] = ra->parts[i * ra->nparts + w];
    }
    prep_tiles += p.prep_tiles_m * p.prep_tiles_n;
    norm[i].partials = reinterpret_cast<const float*>(ws + p.off_partials);
    norm[i].count = p.prep_tiles_m * p.prep_tiles_n;
    norm[i].scale = reinterpret_cast<float*>(ws + p.off_scale);
    const double f = lr_factor(en.m, en.n, hp->lr_adjust);
    apply[i] = make_apply(p, ws, hp->ns_steps, en.param, en.param_dtype, en.update_out, 0,
                          float(1.0 - hp->lr * hp->weight_decay), float(hp->lr * f), apply_tiles);
    apply_tiles += apply[i].tiles_m * apply[i].tiles_n;
  }
  fill_gemm_descs(P, ws, *hp, h);
  const std::vector<double> coeffs = step_coeffs(hp->a, hp->b, hp->c, hp->ns_steps, hp->ns_schedule);
  return enqueue_pipeline(P, ws, slot, hp->ns_steps, coeffs.data(), hp->ns_dtype, hp->momentum,
                          hp->nesterov, hp->eps, prep_tiles, apply_tiles, st, events, ra != nullptr,
                          h);
}

}  // namespace

extern "C" {

size_t mfsdp_ns_workspace_size(int64_t m, int64_t n, int32_t ns_dtype) {
  g_last_error.clear();
  if (!valid_dtype(ns_dtype)) { fail(MFSDP_E_INVALID, "unknown ns_dtype %d", ns_dtype); return 0; }
  if (check_shape(m, n, "matrix", 0)) return 0;
  return make_plan(1, ns_dtype, [&](int64_t, int64_t& mm, int64_t& nn) { mm = m; nn = n; }).bytes;
}

int mfsdp_newton_schulz(const void* x, int32_t x_dtype, void* out, int32_t out_dtype, int64_t m,
                        int64_t n, double a, double b, double c, int32_t steps, double eps,
                        int32_t ns_dtype, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!std::isfinite(a) || !std::isfinite(b) || !std::isfinite(c))
    return fail(MFSDP_E_INVALID, "NS coefficients must be finite");
  if (steps < 0 || steps >= 100) return fail(MFSDP_E_INVALID, "steps must be in [0, 100)");
  const std::vector<double> coeffs = step_coeffs(a, b, c, steps, nullptr);
  return ns_impl(x, x_dtype, out, out_dtype, m, n, coeffs.data(), steps, eps, ns_dtype, workspace,
                 workspace_bytes, stream);
}

int mfsdp_newton_schulz_schedule(const void* x, int32_t x_dtype, void* out, int32_t out_dtype,
                                 int64_t m, int64_t n, const double* coeffs, int32_t steps,
                                 double eps, int32_t ns_dtype, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (steps < 0 || steps >= 100) return fail(MFSDP_E_INVALID, "steps must be in [0, 100)");
  if (steps > 0 && !coeffs) return fail(MFSDP_E_INVALID, "coeffs is NULL");
  for (int i = 0; i < 3 * steps; ++i)
    if (!std::isfinite(coeffs[i])) return fail(MFSDP_E_INVALID, "coeffs entry %d is not finite", i);
  return ns_impl(x, x_dtype, out, out_dtype, m, n, coeffs, steps, eps, ns_dtype, workspace,
                 workspace_bytes, stream);
}

}  // extern "C"

namespace {

// Standalone NS: prep in copy mode (no momentum), the NS products, the output written by the last
// update (bf16) or by the apply pass. coeffs: 3 * steps validated doubles.
int ns_impl(const void* x, int32_t x_dtype, void* out, int32_t out_dtype, int64_t m, int64_t n,
            const double* coeffs, int32_t steps, double eps, int32_t ns_dtype, void* workspace,
            size_t workspace_bytes, void* stream) {
  if (!x || !out) return fail(MFSDP_E_INVALID, "x and out must be non-NULL");
  if (x == out) return fail(MFSDP_E_INVALID, "out must not alias x");
  if (!valid_dtype(x_dtype) || !valid_dtype(out_dtype) || !valid_dtype(ns_dtype))
    return fail(MFSDP_E_INVALID, "unsupported dtype");
  int rc = check_shape(m, n, "matrix", 0);
  if (rc) return rc;
  if (!aligned16(x) || !aligned16(out)) return fail(MFSDP_E_INVALID, "pointers must be 16-byte aligned");
  if (!(eps > 0.0) || !std::isfinite(eps)) return fail(MFSDP_E_INVALID, "eps must be > 0");
  const Plan P = make_plan(1, ns_dtype, [&](int64_t, int64_t& mm, int64_t& nn) { mm = m; nn = n; });
  const DescLayout& dl = P.dl;
  const std::vector<NsPlan>& plans = P.ns;
  const size_t need = P.bytes;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return fail(MFSDP_E_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
  if (workspace_bytes < need)
    return fail(MFSDP_E_WORKSPACE, "workspace too small: %zu < %zu bytes", workspace_bytes, need);

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  void* hptr = nullptr;
  const int slot = ring().acquire(dl.bytes, &hptr, st);
  if (slot < 0) return slot;
  uint8_t* h = static_cast<uint8_t*>(hptr);
  std::memset(h, 0, dl.bytes);
  const NsPlan& p = plans[0];
  auto* prep = reinterpret_cast<PrepDesc*>(h + dl.off_prep);
  auto* norm = reinterpret_cast<NormDesc*>(h + dl.off_norm);
  auto* apply = reinterpret_cast<ApplyDesc*>(h + dl.off_apply);
  prep[0] = make_prep(p, ws, x, x_dtype, nullptr, 0);
  norm[0].partials = reinterpret_cast<const float*>(ws + p.off_partials);
  norm[0].count = p.prep_tiles_m * p.prep_tiles_n;
  norm[0].scale = reinterpret_cast<float*>(ws + p.off_scale);
  apply[0] = make_apply(p, ws, steps, out, out_dtype, nullptr, 1, 1.0f, 0.0f, 0);
  mfsdp_muon_hparams hp{};
  hp.ns_steps = steps;
  hp.ns_dtype = ns_dtype;
  fill_gemm_descs(P, ws, hp, h);
  return enqueue_pipeline(P, ws, slot, steps, coeffs, ns_dtype, 0.0, 0, eps,
                          p.prep_tiles_m * p.prep_tiles_n, apply[0].tiles_m * apply[0].tiles_n, st,
                          nullptr);
}

}  // namespace

extern "C" {

int mfsdp_adamw_step(const mfsdp_adamw_entry* entries, int64_t count, double lr, double beta1,
                     double beta2, double eps, double weight_decay, int64_t step, void* stream) {
  g_last_error.clear();
  if (count < 0) return fail(MFSDP_E_INVALID, "count must be >= 0");
  if (count > 0 && !entries) return fail(MFSDP_E_INVALID, "entries is NULL");
  if (!(lr >= 0.0) || !std::isfinite(lr)) return fail(MFSDP_E_INVALID, "lr must be >= 0");
  if (!(weight_decay >= 0.0) || !std::isfinite(weight_decay))
    return fail(MFSDP_E_INVALID, "weight_decay must be >= 0");
  if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0))
    return fail(MFSDP_E_INVALID, "betas must be in [0, 1)");
  if (!(eps > 0.0) || !std::isfinite(eps)) return fail(MFSDP_E_INVALID, "eps must be > 0");
  if (step < 1) return fail(MFSDP_E_INVALID, "step must be >= 1");
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_adamw_entry& e = entries[i];
    if (!e.param || !e.grad || !e.exp_avg || !e.exp_avg_sq)
      return fail(MFSDP_E_INVALID, "entry %lld: NULL pointer", (long long)i);
    if (e.numel <= 0) return fail(MFSDP_E_INVALID, "entry %lld: numel must be positive", (long long)i);
    if (e.numel > (int64_t(1) << 40)) return fail(MFSDP_E_INVALID, "entry %lld: numel too large", (long long)i);
    if (!valid_dtype(e.param_dtype) || !valid_dtype(e.grad_dtype))
      return fail(MFSDP_E_INVALID, "entry %lld: unsupported dtype", (long long)i);
    if (!aligned16(e.param) || !aligned16(e.grad) || !aligned16(e.exp_avg) || !aligned16(e.exp_avg_sq))
      return fail(MFSDP_E_INVALID, "entry %lld: pointers must be 16-byte aligned", (long long)i);
  }
  if (count == 0) return MFSDP_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const double bc1 = 1.0 - std::pow(beta1, double(step));
  const double bc2 = 1.0 - std::pow(beta2, double(step));
  AdamWBatch batch{};
  batch.decay = float(1.0 - lr * weight_decay);
  batch.beta1 = float(beta1);
  batch.beta2 = float(beta2);
  batch.omb1 = float(1.0 - beta1);
  batch.omb2 = float(1.0 - beta2);
  batch.step_size = float(lr / bc1);
  batch.inv_sqrt_bc2 = float(1.0 / std::sqrt(bc2));
  batch.eps = float(eps);
  int64_t i = 0;
  while (i < count) {
    batch.count = 0;
    int64_t blocks = 0;
    // one launch per group of up to kAdamWMaxPerLaunch tensors; grid kept below 2^31 blocks
    while (i < count && batch.count < kAdamWMaxPerLaunch) {
      const int64_t nb = (entries[i].numel + kAdamWBlockElems - 1) / kAdamWBlockElems;
      if (batch.count > 0 && blocks + nb > (int64_t(1) << 30)) break;
      AdamWDesc& d = batch.d[batch.count++];
      d.param = entries[i].param;
      d.grad = entries[i].grad;
      d.exp_avg = entries[i].exp_avg;
      d.exp_avg_sq = entries[i].exp_avg_sq;
      d.numel = entries[i].numel;
      d.param_dtype = entries[i].param_dtype;
      d.grad_dtype = entries[i].grad_dtype;
      d.block_begin = int32_t(blocks);
      blocks += nb;
      ++i;
    }
    hipError_t e = launch_adamw(batch, int(blocks), st);
    if (e != hipSuccess) return hip_fail(e, "AdamW launch");
  }
  return MFSDP_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------------------------
// Allocation-free Muon step (mfsdp_muon_step_noalloc): its workspace is this static device array,
// one copy per GPU the library runs on, held until the process ends. In host code `scratch` is
// only a host-side stand-in for the symbol; the device address of each GPU's copy comes from
// hipGetSymbolAddress, looked up once per device with that device current and cached here, and
// only that address is handed to kernels. Every call on one GPU shares that GPU's copy.
static __device__ __align__(256) uint8_t scratch[MFSDP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 256;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxScratchDevices] = {};

// Device address of the current device's scratch array (looked up on the first call per device).
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(MFSDP_E_HIP, "device ordinal %d outside [0, %d)", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || (reinterpret_cast<uintptr_t>(p) % kAlign) != 0)
      return fail(MFSDP_E_HIP, "scratch array of device %d is not 256-byte aligned", dev);
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return MFSDP_OK;
}

// Descriptor bytes handed over as kernel arguments, one launch per chunk (vector stores only).
constexpr int kArgChunkWords = 448;  // 1792 bytes of payload per launch
struct ArgChunk {
  uint32_t w[kArgChunkWords];
  uint32_t words;
};

__global__ __launch_bounds__(256) void arg_copy_kernel(ArgChunk c, uint32_t* __restrict__ dst) {
  for (uint32_t i = threadIdx.x; i < c.words; i += blockDim.x) dst[i] = c.w[i];
}

int upload_as_kernel_args(const uint8_t* host, size_t bytes, uint8_t* dst, hipStream_t st) {
  if (bytes % 4) return fail(MFSDP_E_INVALID, "descriptor region of %zu bytes is not whole words", bytes);
  const size_t words = bytes / 4;
  for (size_t w0 = 0; w0 < words; w0 += kArgChunkWords) {
    ArgChunk c;
    c.words = uint32_t(std::min<size_t>(kArgChunkWords, words - w0));
    std::memcpy(c.w, host + 4 * w0, 4 * size_t(c.words));
    hipLaunchKernelGGL(arg_copy_kernel, dim3(1), dim3(256), 0, st, c,
                       reinterpret_cast<uint32_t*>(dst + 4 * w0));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "descriptor launch");
  }
  return MFSDP_OK;
}

}  // namespace

extern "C" int mfsdp_muon_step_noalloc(const mfsdp_muon_entry* entries, int64_t count,
                                       const mfsdp_muon_hparams* hp, void* stream) {
  g_last_error.clear();
  return muon_impl(entries, count, hp, nullptr, 0, stream, nullptr, nullptr, true);
}

namespace mfsdp {
// Descriptor staging shared with the other host modules of the library.
int staging_acquire(size_t bytes, void** host) { return ring().acquire(bytes, host, nullptr); }
int staging_upload(int slot, void* dst, size_t bytes, hipStream_t st) {
  return ring().upload(slot, dst, bytes, st);
}

// One auxiliary stream per device (default priority, non-blocking) and a ring of events for the
// fork / join dependencies between it and the caller's stream, created on first use and kept until
// the process ends. An event may be recorded again while an earlier wait on it is still pending: a
// wait takes the record that precedes it on the host.
namespace {
struct AuxState {
  hipStream_t stream = nullptr;
  hipEvent_t events[8] = {};
  unsigned next = 0;
};
std::mutex g_aux_mu;
std::vector<AuxState> g_aux;
}  // namespace

int aux_stream(hipStream_t* out, hipEvent_t* ev) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lk(g_aux_mu);
  if (dev >= int(g_aux.size())) g_aux.resize(size_t(dev) + 1);
  AuxState& a = g_aux[size_t(dev)];
  if (!a.stream) {
    e = hipStreamCreateWithFlags(&a.stream, hipStreamNonBlocking);
    if (e != hipSuccess) {
      a.stream = nullptr;
      return hip_fail(e, "hipStreamCreateWithFlags");
    }
    for (hipEvent_t& x : a.events) {
      e = hipEventCreateWithFlags(&x, hipEventDisableTiming);
      if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
    }
  }
  *out = a.stream;
  if (ev) *ev = a.events[a.next++ % 8];
  return MFSDP_OK;
}
}  // namespace mfsdp
