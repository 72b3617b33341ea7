// Host side of the Shampoo owner step and of the standalone inverse p-th root: argument checks,
// workspace plan, descriptor build and the launch sequence (all on the caller's stream).
//
// Shampoo (Section 5.7 of the paper; Gupta, Koren and Singer 2018, matrix case) per owned matrix:
//   L <- beta L + weight G G^T,  R <- beta R + weight G^T G
//   refresh: P_L = (L + rho_L I)^(-1/4), P_R = (R + rho_R I)^(-1/4), rho = eps + eps_rel ||S||_F
//   U = P_L G P_R,  p <- p (1 - lr wd) - lr U
//
// Convergence: the M product of every iteration also records max |M - I| over the real block; once
// it is below kShConvTol, the side's later products are skipped and its X products become copies.
//
// Inverse p-th root by the coupled Newton iteration (Guo and Higham, SIAM J. Matrix Anal. Appl.
// 2006; the form used for Shampoo by Anil et al. 2020): with z = (1 + p) / (2 ||A||_F),
//   X_0 = z^(1/p) I,  M_0 = z A,  T_k = ((p + 1) I - M_k) / p,
//   X_{k+1} = X_k T_k,  M_{k+1} = T_k^p M_k,
// so that M_k -> I and X_k -> A^(-1/p). All iterates are polynomials in A, hence symmetric and
// commuting: every product is an NT product of symmetric operands, computed on its upper tiles.
// T_k is never stored; its affine form is folded into the products:
//   X_{k+1}  = ((p+1)/p) X_k - (1/p) X_k M_k
//   T_k^2    = (p+1)^2/p^2 I - 2(p+1)/p^2 M_k + 1/p^2 M_k M_k
//   T_k^4    = T_k^2 T_k^2,   M_{k+1} = T_k^p M_k          (p = 1: M_{k+1} = 2 M_k - M_k M_k)
// The last iteration forms X only.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "shampoo_build.h"

using namespace mfsdp;
using namespace mfsdp::shb;

namespace {

constexpr int kNormChunkRows = 16;
constexpr int64_t kMaxDim = 1 << 16;

// One inverse-root problem on a padded d_pad x d_pad statistic, held in M or, when S is set, at S
// (a caller buffer, row stride d_pad; M then only receives the iteration's first M).
struct Side {
  int64_t d = 0, dp = 0;
  size_t M = 0, T2 = 0, T4 = 0, X[2] = {0, 0}, partials = 0, sc = 0, resid = 0;
  const float* S = nullptr;
  float* out = nullptr;  // caller destination of the root (d x d, row stride d)
  bool has_out = false;  // copy the root out (decided by the call, not by the pointer value,
                         // so that the size query, which sees no pointers, builds the same ops)
};

void plan_side(Side& s, int64_t d, Arena& a) {
  s.d = d;
  s.dp = rup(d, kShTile);
  const size_t mat = size_t(s.dp) * size_t(s.dp) * sizeof(float);
  s.M = a.take(mat);
  s.T2 = a.take(mat);
  s.T4 = a.take(mat);
  s.X[0] = a.take(mat);
  s.X[1] = a.take(mat);
  s.partials = a.take(size_t(s.dp / kNormChunkRows) * 2 * sizeof(double));
  s.sc = a.take(4 * sizeof(float));
  s.resid = a.take(2 * sizeof(float));
}

// Gp, GpT: G and G^T zero-padded (fp32, or for a bf16 gradient bf16 G and G^T both in Gp, which
// leaves GpT free); Y = P_L G (or Y^T = P_R G^T for a wide bf16 G); U goes to Gp for an fp32
// gradient, GpT for a bf16 one.
struct EntryPlan {
  int64_t m, n, mp, np;
  bool grad_bf16;
  size_t Gp, GpT, Y;
  Side L, R;
  size_t g() const { return Gp; }  // G (row stride np)
  size_t gt() const {              // G^T (row stride mp)
    return grad_bf16 ? Gp + size_t(mp) * size_t(np) * 2 : GpT;
  }
  size_t u() const { return grad_bf16 ? GpT : Gp; }
};

// Root ops for every side: norms, scalars, init, the iterations and the copy of X to side.out.
// In every grouped launch the larger problems come first (their tiles run longest), so the
// hardware's in-order dispatch fills the tail of the launch with the short tiles.
void add_root_ops(Build& b, std::vector<Side*> sides, int p, int iters) {
  std::stable_sort(sides.begin(), sides.end(), [](const Side* x, const Side* y) { return x->dp > y->dp; });
  std::vector<ShNormDesc> nd;
  std::vector<ShScalarDesc> sd;
  std::vector<ShInitDesc> idesc;
  int nblocks = 0, itiles = 0;
  for (Side* s : sides) {
    ShNormDesc n{};
    n.S = s->S ? s->S : b.ptr<float>(s->M);
    n.ld = s->dp;
    n.rows_pad = int32_t(s->dp);
    n.chunk_rows = kNormChunkRows;
    n.partials = b.ptr<double>(s->partials);
    n.nchunks = int32_t(s->dp / kNormChunkRows);
    n.tile_begin = nblocks;
    nblocks += n.nchunks;
    nd.push_back(n);
    ShScalarDesc c{};
    c.partials = n.partials;
    c.nchunks = n.nchunks;
    c.d = int32_t(s->d);
    c.out = b.ptr<float>(s->sc);
    sd.push_back(c);
    ShInitDesc in{};
    in.S = n.S;
    in.M = b.ptr<float>(s->M);
    in.X = b.ptr<float>(s->X[0]);
    in.resid = b.ptr<float>(s->resid);
    in.ld = s->dp;
    in.sc = c.out;
    in.tiles_n = int32_t(s->dp / kShCopyTile);
    in.tile_begin = itiles;
    itiles += int((s->dp / kShCopyTile) * (s->dp / kShCopyTile));
    idesc.push_back(in);
  }
  b.op(kOpNorm, nd, nblocks);
  b.op(kOpScalars, sd, int(sd.size()));
  b.op(kOpInit, idesc, itiles);

  const float fp = float(p);
  // per parity q: A holds M_k, B receives M_{k+1}; X[q] -> X[q ^ 1]; residual slots q^1 (read)
  // and q (cleared by the first launch of the iteration, written by the M product)
  std::vector<ShGemmDesc> l1[2], l2[2], l3[2];
  int t1[2] = {0, 0}, t1x[2] = {0, 0}, t2[2] = {0, 0}, t3[2] = {0, 0};
  auto roots = [&](ShGemmDesc g, const Side* s, int q) {
    g.conv_in = b.ptr<float>(s->resid + sizeof(float) * (q ^ 1));
    g.valid = int32_t(s->d);
    return g;
  };
  for (int q = 0; q < 2; ++q) {
    for (Side* s : sides) {  // X products first, so the last iteration launches a prefix
      const int64_t dp = s->dp;
      float* A = b.ptr<float>(q == 0 ? s->M : s->T2);
      ShGemmDesc g = roots(gemm_desc(b.ptr<float>(s->X[q]), A, b.ptr<float>(s->X[q]),
                                     b.ptr<float>(s->X[q ^ 1]), dp, dp, dp, dp, dp, dp, dp, 1,
                                     -1.0f / fp, (fp + 1.0f) / fp, 0.0f, t1[q]), s, q);
      g.copy_on_skip = 1;
      g.clear = b.ptr<float>(s->resid + sizeof(float) * q);
      l1[q].push_back(g);
    }
    t1x[q] = t1[q];
    for (Side* s : sides) {
      const int64_t dp = s->dp;
      float* A = b.ptr<float>(q == 0 ? s->M : s->T2);
      float* B = b.ptr<float>(q == 0 ? s->T2 : s->M);
      float* T4 = b.ptr<float>(s->T4);
      ShGemmDesc mupd;
      if (p == 1) {
        mupd = roots(gemm_desc(A, A, A, B, dp, dp, dp, dp, dp, dp, dp, 1, -1.0f, 2.0f, 0.0f, t3[q]), s, q);
      } else {
        const float ip2 = 1.0f / (fp * fp);
        l1[q].push_back(roots(gemm_desc(A, A, A, p == 4 ? B : T4, dp, dp, dp, dp, dp, dp, dp, 1, ip2,
                                        -2.0f * (fp + 1.0f) * ip2, (fp + 1.0f) * (fp + 1.0f) * ip2, t1[q]),
                              s, q));
        if (p == 4)
          l2[q].push_back(roots(gemm_desc(B, B, nullptr, T4, dp, dp, 0, dp, dp, dp, dp, 1, 1.0f, 0.0f, 0.0f,
                                          t2[q]), s, q));
        mupd = roots(gemm_desc(T4, A, nullptr, B, dp, dp, 0, dp, dp, dp, dp, 1, 1.0f, 0.0f, 0.0f, t3[q]), s, q);
      }
      mupd.resid_out = b.ptr<float>(s->resid + sizeof(float) * q);
      l3[q].push_back(mupd);
    }
  }
  size_t o1[2], o2[2] = {0, 0}, o3[2] = {0, 0};
  for (int q = 0; q < 2; ++q) {
    o1[q] = b.put(l1[q]);
    if (!l2[q].empty()) o2[q] = b.put(l2[q]);
    if (!l3[q].empty()) o3[q] = b.put(l3[q]);
  }
  const int ns = int(sides.size());
  for (int k = 0; k < iters; ++k) {
    const int q = k & 1;
    const bool last = k == iters - 1;
    b.ops.push_back(Op{kOpGemm, o1[q], last ? ns : int(l1[q].size()), last ? t1x[q] : t1[q]});
    if (last) break;
    if (!l2[q].empty()) b.ops.push_back(Op{kOpGemm, o2[q], int(l2[q].size()), t2[q]});
    if (!l3[q].empty()) b.ops.push_back(Op{kOpGemm, o3[q], int(l3[q].size()), t3[q]});
  }
  std::vector<ShCopyDesc> co;
  int ct = 0;
  for (Side* s : sides) {
    if (!s->has_out) continue;
    co.push_back(copy_desc(b.ptr<float>(s->X[iters & 1]), kDtF32, s->out, nullptr, s->d, s->d, s->dp,
                           s->d, 0, s->d, s->d, ct));
  }
  b.op(kOpCopyOut, co, ct);
}

int check_shampoo_hp(const mfsdp_shampoo_hparams* hp) {
  if (!hp) return bad("hparams is NULL");
  auto fin = [](double x) { return std::isfinite(x); };
  if (!(hp->lr >= 0.0) || !fin(hp->lr)) return bad("lr must be finite and >= 0");
  if (!(hp->weight_decay >= 0.0) || !fin(hp->weight_decay)) return bad("weight_decay must be finite and >= 0");
  if (!(hp->beta >= 0.0) || !fin(hp->beta)) return bad("beta must be finite and >= 0");
  if (!(hp->weight >= 0.0) || !fin(hp->weight)) return bad("weight must be finite and >= 0");
  if (!(hp->eps > 0.0) || !fin(hp->eps)) return bad("eps must be finite and > 0");
  if (!(hp->eps_rel >= 0.0) || !fin(hp->eps_rel)) return bad("eps_rel must be finite and >= 0");
  if (hp->refresh != 0 && hp->refresh != 1) return bad("refresh must be 0 or 1");
  if (hp->root_iters < 1 || hp->root_iters > 100) return bad("root_iters must be in [1, 100]");
  return MFSDP_OK;
}

int check_shampoo_entries(const mfsdp_shampoo_entry* en, int64_t count, bool data) {
  if (count < 0) return bad("count must be >= 0");
  if (count > 0 && !en) return bad("entries is NULL");
  if (count > 4096) return bad("at most 4096 entries per call");
  int64_t units = 0;  // bound on the 64 x 64 tiles of any one grouped launch (grid and int32 counters)
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_shampoo_entry& e = en[i];
    const std::string w = "entry " + std::to_string(i) + ": ";
    if (e.m < 1 || e.n < 1 || e.m > kMaxDim || e.n > kMaxDim) return bad(w + "m and n must be in [1, 65536]");
    const int64_t s = rup(e.m, kShTile) + rup(e.n, kShTile);
    units += 3 * (s / kShCopyTile) * (s / kShCopyTile);
    if (units > (int64_t(1) << 30)) return bad("the entries of one call exceed 2^30 tiles per launch");
    if (!dtype_ok(e.param_dtype) || !dtype_ok(e.grad_dtype)) return bad(w + "dtype must be F32 or BF16");
    if (!data) continue;
    if (!e.param || !e.grad || !e.L || !e.R || !e.PL || !e.PR) return bad(w + "NULL pointer");
    const size_t pa = e.param_dtype == MFSDP_BF16 ? 2 : 4, ga = e.grad_dtype == MFSDP_BF16 ? 2 : 4;
    if (!aligned(e.param, pa) || !aligned(e.grad, ga) || !aligned(e.L, 4) || !aligned(e.R, 4) ||
        !aligned(e.PL, 4) || !aligned(e.PR, 4) || !aligned(e.update_out, 4))
      return bad(w + "misaligned pointer");
  }
  return MFSDP_OK;
}

// Builds the whole Shampoo step for `count` entries. Returns the workspace bytes (buffers, then
// the descriptor region at desc_at). `sizing`: for the size query, which sees no pointers (every
// side is then taken as copied: the most descriptors a step can need).
size_t build_shampoo(const mfsdp_shampoo_entry* en, int64_t count, const mfsdp_shampoo_hparams* hp,
                     char* ws, Build& b, size_t& desc_at, bool sizing) {
  b.base = ws;
  Arena a;
  std::vector<EntryPlan> P(static_cast<size_t>(count));
  for (int64_t i = 0; i < count; ++i) {
    EntryPlan& e = P[size_t(i)];
    e.m = en[i].m;
    e.n = en[i].n;
    e.mp = rup(e.m, kShTile);
    e.np = rup(e.n, kShTile);
    e.grad_bf16 = en[i].grad_dtype == MFSDP_BF16;
    const size_t gbytes = size_t(e.mp) * size_t(e.np) * sizeof(float);
    e.Gp = a.take(gbytes);
    e.GpT = a.take(gbytes);
    e.Y = a.take(gbytes);
    plan_side(e.L, e.m, a);
    plan_side(e.R, e.n, a);
    e.L.out = en[i].PL;
    e.R.out = en[i].PR;
    e.L.has_out = e.R.has_out = true;
    // a side whose dimension is a multiple of the tile works on the caller's buffers where they
    // lie (their layout is the padded one; 16-byte aligned, as the GEMM's vector accesses need):
    // the statistic is updated in place and the root is taken of it there, a stored
    // preconditioner is read there; neither is copied in or out
    if (!sizing && e.m == e.mp && aligned(en[i].L, 16) && aligned(en[i].PL, 16)) e.L.S = en[i].L;
    if (!sizing && e.n == e.np && aligned(en[i].R, 16) && aligned(en[i].PR, 16)) e.R.S = en[i].R;
  }
  desc_at = a.off;
  const bool refresh = hp->refresh != 0;
  const int iters = hp->root_iters;
  const int fin = refresh ? (iters & 1) : 0;

  std::vector<ShCopyDesc> cin;
  int ct = 0;
  for (int64_t i = 0; i < count; ++i) {
    EntryPlan& e = P[size_t(i)];
    // a bf16 gradient is copied as bf16 (exact): the GEMM reads it as a one-part operand
    cin.push_back(copy_desc(en[i].grad, en[i].grad_dtype, b.ptr<float>(e.g()), b.ptr<float>(e.gt()), e.m, e.n,
                            e.n, e.np, e.mp, e.mp, e.np, ct));
    cin.back().dst_bf16 = e.grad_bf16 ? 1 : 0;
    if (!e.L.S)
      cin.push_back(copy_desc(en[i].L, kDtF32, b.ptr<float>(e.L.M), nullptr, e.m, e.m, e.m, e.mp, 0, e.mp,
                              e.mp, ct));
    if (!e.R.S)
      cin.push_back(copy_desc(en[i].R, kDtF32, b.ptr<float>(e.R.M), nullptr, e.n, e.n, e.n, e.np, 0, e.np,
                              e.np, ct));
    if (!refresh && !e.L.S)
      cin.push_back(copy_desc(en[i].PL, kDtF32, b.ptr<float>(e.L.X[0]), nullptr, e.m, e.m, e.m, e.mp, 0,
                              e.mp, e.mp, ct));
    if (!refresh && !e.R.S)
      cin.push_back(copy_desc(en[i].PR, kDtF32, b.ptr<float>(e.R.X[0]), nullptr, e.n, e.n, e.n, e.np, 0,
                              e.np, e.np, ct));
  }
  b.op(kOpCopyIn, cin, ct);

  // grouped products over the entries, largest first (see add_root_ops)
  std::vector<EntryPlan*> order;
  for (auto& e : P) order.push_back(&e);
  std::stable_sort(order.begin(), order.end(), [](const EntryPlan* x, const EntryPlan* y) {
    return std::max(x->mp, x->np) > std::max(y->mp, y->np);
  });
  // a bf16 gradient is one bf16 part: the statistics take one product, P_L G three
  auto stat = [&](const Side& s, float* caller) { return s.S ? caller : b.ptr<float>(s.M); };
  std::vector<ShGemmDesc> gs;
  int gt = 0;
  for (EntryPlan* ep : order) {
    EntryPlan& e = *ep;
    const mfsdp_shampoo_entry& c = en[ep - P.data()];
    const int bf = e.grad_bf16 ? 1 : 0;
    float* Ls = stat(e.L, c.L);
    float* Rs = stat(e.R, c.R);
    gs.push_back(gemm_desc(b.ptr<float>(e.g()), b.ptr<float>(e.g()), Ls, Ls, e.np, e.np, e.mp, e.mp, e.mp, e.mp,
                           e.np, 1, float(hp->weight), float(hp->beta), 0.0f, gt));
    gs.back().p_bf16 = gs.back().q_bf16 = bf;
    gs.push_back(gemm_desc(b.ptr<float>(e.gt()), b.ptr<float>(e.gt()), Rs, Rs, e.mp, e.mp, e.np, e.np, e.np, e.np,
                           e.mp, 1, float(hp->weight), float(hp->beta), 0.0f, gt));
    gs.back().p_bf16 = gs.back().q_bf16 = bf;
  }
  b.op(kOpGemm, gs, gt);

  std::vector<ShCopyDesc> cst;
  ct = 0;
  for (int64_t i = 0; i < count; ++i) {
    EntryPlan& e = P[size_t(i)];
    if (!e.L.S)
      cst.push_back(copy_desc(b.ptr<float>(e.L.M), kDtF32, en[i].L, nullptr, e.m, e.m, e.mp, e.m, 0, e.m,
                              e.m, ct));
    if (!e.R.S)
      cst.push_back(copy_desc(b.ptr<float>(e.R.M), kDtF32, en[i].R, nullptr, e.n, e.n, e.np, e.n, 0, e.n,
                              e.n, ct));
  }
  b.op(kOpCopyOut, cst, ct);

  if (refresh) {
    std::vector<Side*> sides;
    for (auto& e : P) {
      sides.push_back(&e.L);
      sides.push_back(&e.R);
    }
    add_root_ops(b, sides, 4, iters);
  }

  std::vector<ShGemmDesc> gy, gu;
  int ty = 0, tu = 0;
  for (EntryPlan* ep : order) {
    EntryPlan& e = *ep;
    const size_t i = size_t(ep - P.data());
    // the preconditioners: this step's roots, or the stored ones (read where they lie, or copied)
    const float* pl = (!refresh && e.L.S) ? en[i].PL : b.ptr<float>(e.L.X[fin]);
    const float* pr = (!refresh && e.R.S) ? en[i].PR : b.ptr<float>(e.R.X[fin]);
    // U = P_L G P_R^T. Both association orders take the same fp32 flop, but with a bf16 G the product
    // that reads G takes three bf16 MFMAs per step and the other six, so the larger of the two
    // products should be the one with G: a wide G (n > m) forms Y^T = P_R G^T (n x m) first and then
    // U = P_L Y; otherwise Y = P_L G, then U = Y P_R^T.
    if (e.grad_bf16 && e.n > e.m) {
      gy.push_back(gemm_desc(pr, b.ptr<float>(e.g()), nullptr, b.ptr<float>(e.Y), e.np, e.np, 0, e.mp, e.np,
                             e.mp, e.np, 0, 1.0f, 0.0f, 0.0f, ty));
      gy.back().q_bf16 = 1;
      gu.push_back(gemm_desc(pl, b.ptr<float>(e.Y), nullptr, b.ptr<float>(e.u()), e.mp, e.mp, 0, e.np, e.mp,
                             e.np, e.mp, 0, 1.0f, 0.0f, 0.0f, tu));
    } else {
      gy.push_back(gemm_desc(pl, b.ptr<float>(e.gt()), nullptr, b.ptr<float>(e.Y), e.mp, e.mp, 0, e.np, e.mp,
                             e.np, e.mp, 0, 1.0f, 0.0f, 0.0f, ty));
      gy.back().q_bf16 = e.grad_bf16 ? 1 : 0;
      gu.push_back(gemm_desc(b.ptr<float>(e.Y), pr, nullptr, b.ptr<float>(e.u()), e.np, e.np, 0, e.np, e.mp,
                             e.np, e.np, 0, 1.0f, 0.0f, 0.0f, tu));
    }
  }
  b.op(kOpGemm, gy, ty);
  b.op(kOpGemm, gu, tu);

  std::vector<ShApplyDesc> ap;
  int at = 0;
  for (int64_t i = 0; i < count; ++i) {
    EntryPlan& e = P[size_t(i)];
    ShApplyDesc d{};
    d.U = b.ptr<float>(e.u());
    d.ldu = e.np;
    d.param = en[i].param;
    d.update_out = en[i].update_out;
    d.m = e.m;
    d.n = e.n;
    d.param_dtype = en[i].param_dtype == MFSDP_BF16 ? kDtBF16 : kDtF32;
    const int64_t tn = (e.n + kShCopyTile - 1) / kShCopyTile, tm = (e.m + kShCopyTile - 1) / kShCopyTile;
    d.tiles_n = int32_t(tn);
    d.tile_begin = at;
    at += int(tm * tn);
    ap.push_back(d);
  }
  b.op(kOpApply, ap, at);
  return desc_at + al(b.h.size());
}

size_t build_root(int64_t d, int p, int iters, const float* a, float* out, char* ws, Build& b,
                  size_t& desc_at, bool sizing) {
  b.base = ws;
  Arena ar;
  Side s;
  plan_side(s, d, ar);
  s.out = out;
  s.has_out = true;
  desc_at = ar.off;
  if (!sizing && d == s.dp && aligned(a, 16)) {
    s.S = a;  // read where it lies
  } else {
    std::vector<ShCopyDesc> cin;
    int ct = 0;
    cin.push_back(copy_desc(a, kDtF32, b.ptr<float>(s.M), nullptr, d, d, d, s.dp, 0, s.dp, s.dp, ct));
    b.op(kOpCopyIn, cin, ct);
  }
  std::vector<Side*> sides{&s};
  add_root_ops(b, sides, p, iters);
  return desc_at + al(b.h.size());
}

}  // namespace

extern "C" {

size_t mfsdp_shampoo_workspace_size(const mfsdp_shampoo_entry* entries, int64_t count,
                                    const mfsdp_shampoo_hparams* hp) {
  if (check_shampoo_entries(entries, count, false) != MFSDP_OK) return 0;
  if (check_shampoo_hp(hp) != MFSDP_OK) return 0;
  if (count == 0) return 0;
  Build b;
  size_t desc_at = 0;
  return build_shampoo(entries, count, hp, nullptr, b, desc_at, true);
}

int mfsdp_shampoo_step(const mfsdp_shampoo_entry* entries, int64_t count, const mfsdp_shampoo_hparams* hp,
                       void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_shampoo_entries(entries, count, true);
  if (rc != MFSDP_OK) return rc;
  rc = check_shampoo_hp(hp);
  if (rc != MFSDP_OK) return rc;
  if (count == 0) return MFSDP_OK;
  Build b;
  size_t desc_at = 0;
  const size_t need = build_shampoo(entries, count, hp, static_cast<char*>(workspace), b, desc_at, false);
  if (!workspace || !aligned(workspace, kAl) || workspace_bytes < need)
    return set_last_error(MFSDP_E_WORKSPACE, "workspace NULL, not 256-byte aligned or smaller than "
                                             "mfsdp_shampoo_workspace_size (" + std::to_string(need) + " bytes)");
  RunScalars rs;
  rs.eps = hp->eps;
  rs.eps_rel = hp->eps_rel;
  rs.p = 4;
  rs.decay = float(1.0 - hp->lr * hp->weight_decay);
  rs.step = float(hp->lr);
  return run(b, static_cast<char*>(workspace), desc_at, static_cast<hipStream_t>(stream), rs);
}

size_t mfsdp_inverse_root_workspace_size(int64_t d, int32_t p, int32_t iters) {
  if (d < 1 || d > kMaxDim || (p != 1 && p != 2 && p != 4) || iters < 1 || iters > 100) return 0;
  Build b;
  size_t desc_at = 0;
  return build_root(d, p, iters, nullptr, nullptr, nullptr, b, desc_at, true);
}

int mfsdp_inverse_root(const float* a, float* out, int64_t d, int32_t p, double eps, double eps_rel,
                       int32_t iters, void* workspace, size_t workspace_bytes, void* stream) {
  if (!a || !out) return bad("a and out must be non-NULL");
  if (!aligned(a, 4) || !aligned(out, 4)) return bad("misaligned pointer");
  if (d < 1 || d > kMaxDim) return bad("d must be in [1, 65536]");
  if (p != 1 && p != 2 && p != 4) return bad("p must be 1, 2 or 4");
  if (!(eps > 0.0) || !std::isfinite(eps)) return bad("eps must be finite and > 0");
  if (!(eps_rel >= 0.0) || !std::isfinite(eps_rel)) return bad("eps_rel must be finite and >= 0");
  if (iters < 1 || iters > 100) return bad("iters must be in [1, 100]");
  Build b;
  size_t desc_at = 0;
  const size_t need = build_root(d, p, iters, a, out, static_cast<char*>(workspace), b, desc_at, false);
  if (!workspace || !aligned(workspace, kAl) || workspace_bytes < need)
    return set_last_error(MFSDP_E_WORKSPACE, "workspace NULL, not 256-byte aligned or smaller than "
                                             "mfsdp_inverse_root_workspace_size (" + std::to_string(need) + " bytes)");
  RunScalars rs;
  rs.eps = eps;
  rs.eps_rel = eps_rel;
  rs.p = p;
  return run(b, static_cast<char*>(workspace), desc_at, static_cast<hipStream_t>(stream), rs);
}

}  // extern "C"
