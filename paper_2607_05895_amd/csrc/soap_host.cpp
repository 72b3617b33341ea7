// Host side of the SOAP owner step and of the standalone orthonormal factor: argument checks,
// workspace plan, descriptor build and the launch sequence (all on the caller's stream).
//
// SOAP (Section 5.7 of the paper: Adam in the eigenbasis of Shampoo's statistics; Vyas et al. 2024,
// matrix case) per owned m x n matrix, with the bases Q_L, Q_R of the previous refresh:
//   G' = Q_L^T G Q_R,  M <- beta1 M + (1 - beta1) G,  M' = Q_L^T M Q_R
//   V <- beta2 V + (1 - beta2) G'^2,  N' = bias-corrected M' / (sqrt(V) + eps),  N = Q_L N' Q_R^T
//   p <- p (1 - lr wd) - lr N;  L <- beta_s L + w_s G G^T, R <- beta_s R + w_s G^T G
//   refresh: Q_L <- Q of QR(L Q_L), Q_R <- Q of QR(R Q_R)   (refresh_iters times)
//
// Every product is an NT product C = alpha P Q^T (+ beta E) on the Shampoo GEMM, over padded
// row-major buffers (mp, np = m, n rounded up to 128), grouped over the entries:
//   X1      = Q_L^T [G | M]      P = Q_L^T,  Q = [G^T ; M^T]        (two mp x np, K = mp)
//   [G'|M'] = X1 halves . Q_R    P = X1 half, Q = Q_R^T              (two mp x np, K = np)
//   Z       = Q_L N'             P = Q_L,    Q = N'^T               (mp x np, K = mp)
//   N       = Z Q_R^T            P = Z,      Q = Q_R                (mp x np, K = np)
//   L, R statistics              P = Q = G (sym, K = np), P = Q = G^T (sym, K = mp)
//   refresh S^T = Q_L^T L        P = Q_L^T,  Q = L                  (mp x mp, K = mp)
// A bf16 gradient is kept as bf16 (G, and the G^T half of [G^T ; M^T]) and is a one-part operand
// of the split-bf16 GEMM: the statistics then take one bf16 product per step, Q_L^T G three. For a
// wide matrix (n > m) with both bases the right product runs first (X1 = Q_R^T [G^T | M^T] with G
// and M read row-major, then [G' | M'] = Q_L^T X1^T), so that the larger product is the one with
// the one-part G.
// The first-moment pass writes G, G^T and M^T; the Adam pass writes N'^T; both bases are copied in
// with their transposes. The refresh QR is a blocked Householder factorization of S's real d x d
// block, with S held transposed (each column of S one contiguous row) and Q accumulated from the
// identity as Q <- Q H_B per 128-column block B. Per block: eight 16-column panel launches (the
// panel's reflectors), each but the last followed by a launch that applies them to the block's
// later columns (one workgroup per column); then on the Shampoo GEMM G = V^T V (K-split) with
// W = X V, the block's T (one workgroup), U = V T^T and X <- X - W U^T for X = the trailing columns
// of S (as rows of S^T) and X = Q's columns [j0, dp). The part of that update beyond the next
// block's columns runs on an auxiliary stream, overlapping the next block's panels (look-ahead).
// Zero padding is exact: padded rows and columns of G, M, the bases and the statistics are zero, so
// every product's real block is unaffected and its padded part is zero.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "shampoo_build.h"

using namespace mfsdp;
using namespace mfsdp::shb;

namespace {

// One basis refresh problem: St (dp x dp) holds S^T (real block d x d) and is factored in place; Q
// (dp x dp) accumulates the orthonormal factor (row-major, zero padding). V, Vt, T, G, U, Ws, Wq hold
// the current block's reflectors, factor and products.
struct QrSide {
  int64_t d = 0, dp = 0;
  size_t St = 0, Q = 0, V = 0, Vt = 0, T = 0, G = 0, U = 0, Ws = 0, Wq = 0;
};

constexpr int64_t kQrMaxGram = (kQrMaxDim + kQrGramChunk - 1) / kQrGramChunk;  // partials of V^T V

void plan_qr_buffers(QrSide& s, Arena& a) {
  const size_t f = sizeof(float), col = size_t(s.dp) * kQrBlock * f, sq = size_t(kQrBlock) * kQrBlock * f;
  s.V = a.take(col);
  s.Vt = a.take(col);
  s.U = a.take(col);
  s.Ws = a.take(col);
  s.Wq = a.take(col);
  s.T = a.take(sq);
  s.G = a.take(size_t(kQrMaxGram) * sq);
}

// A grouped product before its tile offset is known (so that a launch can be ordered by cost).
struct Prod {
  const float *P, *Q, *E;
  float* C;
  int64_t ldp, ldq, lde, ldc, M, N, K;
  int sym;
  float alpha, beta;
  bool pbf = false, qbf = false;  // P, Q stored as bf16 (one-part operands; both, or Q alone)
};

void add_gemm(Build& b, std::vector<Prod> ps) {
  // longest tiles first (K times the bf16 products per step; a one-part product is load-bound at
  // about a third of the six-product time): the hardware dispatches blocks in order
  auto cost = [](const Prod& x) { return x.K * (x.pbf && x.qbf ? 2 : x.qbf ? 3 : 6); };
  std::stable_sort(ps.begin(), ps.end(), [&](const Prod& x, const Prod& y) { return cost(x) > cost(y); });
  std::vector<ShGemmDesc> gs;
  int gt = 0;
  for (const Prod& p : ps) {
    gs.push_back(gemm_desc(p.P, p.Q, p.E, p.C, p.ldp, p.ldq, p.lde, p.ldc, p.M, p.N, p.K, p.sym, p.alpha,
                           p.beta, 0.0f, gt));
    gs.back().p_bf16 = p.pbf ? 1 : 0;
    gs.back().q_bf16 = p.qbf ? 1 : 0;
  }
  b.op(kOpGemm, gs, gt);
}

// The block update's products for each side, over X = the trailing columns of S (rows [j0 + 128,
// dp) of St) and X = Q's columns [j0, dp): kW appends W = X V (whole X) to ps; kXNext appends
// X <- X - W U^T for St's next 128 rows (the next block's columns); kXRest appends it for the
// remaining St rows and for Q.
enum WxPart { kW, kXNext, kXRest };
void add_wx(Build& b, const std::vector<QrSide*>& act, int64_t j0, WxPart part, std::vector<Prod>& ps) {
  for (QrSide* s : act) {
    const int64_t vrows = s->dp - j0;
    const float* Vt = b.ptr<float>(s->Vt);
    const float* U = b.ptr<float>(s->U);
    const int64_t trail = s->dp - j0 - kQrBlock;  // St rows [j0 + 128, dp)
    const bool has_trail = trail > 0 && j0 + kQrBlock < s->d;
    float* XS = b.ptr<float>(s->St) + (j0 + kQrBlock) * s->dp + j0;
    float* WS = b.ptr<float>(s->Ws);
    float* XQ = b.ptr<float>(s->Q) + j0;
    float* WQ = b.ptr<float>(s->Wq);
    auto w = [&](float* X, float* W, int64_t rows) {
      ps.push_back(Prod{X, Vt, nullptr, W, s->dp, s->dp, 0, kQrBlock, rows, kQrBlock, vrows, 0, 1.0f, 0.0f});
    };
    auto x = [&](float* X, const float* W, int64_t rows) {
      ps.push_back(Prod{W, U, X, X, kQrBlock, kQrBlock, s->dp, s->dp, rows, vrows, kQrBlock, 0, -1.0f, 1.0f});
    };
    if (part == kW) {
      if (has_trail) w(XS, WS, trail);
      w(XQ, WQ, s->dp);
    } else if (part == kXNext) {
      if (has_trail) x(XS, WS, kQrBlock);
    } else {
      if (has_trail && trail > kQrBlock)
        x(XS + kQrBlock * s->dp, WS + kQrBlock * kQrBlock, trail - kQrBlock);
      x(XQ, WQ, s->dp);
    }
  }
}

// The Householder QR of each side's S (given as St): Q = H_1 H_2 ... H_d into each side's Q buffer
// (set to the identity first). Sides are listed largest first in every grouped launch.
void add_qr_ops(Build& b, std::vector<QrSide*> sides) {
  if (sides.empty()) return;
  std::stable_sort(sides.begin(), sides.end(), [](const QrSide* x, const QrSide* y) { return x->d > y->d; });
  {
    std::vector<SoapEyeDesc> ey;
    int et = 0;
    for (QrSide* s : sides) {
      SoapEyeDesc e{};
      e.X = b.ptr<float>(s->Q);
      e.ld = s->dp;
      e.d = s->d;
      e.dp = s->dp;
      const int64_t tn = s->dp / kShCopyTile;
      e.tiles_n = int32_t(tn);
      e.tile_begin = et;
      et += int(tn * tn);
      ey.push_back(e);
    }
    b.op(kOpEye, ey, et);
  }
  for (int64_t j0 = 0; j0 < sides[0]->d; j0 += kQrBlock) {
    std::vector<QrSide*> act;
    for (QrSide* s : sides)
      if (s->d > j0) act.push_back(s);
    // panels and their application to the rest of the block
    for (int64_t c = j0; c < j0 + kQrBlock; c += kQrPanel) {
      std::vector<QrPanelDesc> pd;
      std::vector<QrColDesc> cd;
      int ct = 0;
      for (QrSide* s : act) {
        QrPanelDesc p{};
        p.At = b.ptr<float>(s->St);
        p.ld = s->dp;
        p.V = b.ptr<float>(s->V);
        p.Vt = b.ptr<float>(s->Vt);
        p.T = b.ptr<float>(s->T);
        p.ldvt = s->dp;
        p.j0 = int32_t(j0);
        p.c = int32_t(c);
        p.jb = int32_t(std::clamp<int64_t>(s->d - c, 0, kQrPanel));
        p.d = int32_t(s->d);
        p.vrows = int32_t(s->dp - j0);
        pd.push_back(p);
        const int64_t ncols = std::min(j0 + kQrBlock, s->d) - (c + kQrPanel);
        if (ncols > 0) {
          QrColDesc q{};
          q.At = b.ptr<float>(s->St);
          q.ld = s->dp;
          q.V = b.ptr<float>(s->V) + (c - j0) * kQrBlock + (c - j0);
          q.T = b.ptr<float>(s->T) + (c - j0) * kQrBlock + (c - j0);
          q.c = int32_t(c);
          q.rows = int32_t(s->d - c);
          q.ncols = int32_t(ncols);
          q.tile_begin = ct;
          ct += int(ncols);
          cd.push_back(q);
        }
      }
      b.op(kOpQrPanel, pd, int(pd.size()));
      if (!cd.empty()) b.op(kOpQrCol, cd, ct);
    }
    // (the previous block's update of the trailing columns beyond this block and of Q, on the
    // auxiliary stream, overlapped the panels above; it must end before W reads them)
    if (j0 > 0) b.join();
    // G = V^T V in K chunks together with W = X V (both read only V), then the block's T
    {
      std::vector<Prod> gp;
      std::vector<QrTDesc> td;
      for (QrSide* s : act) {
        const int64_t vrows = s->dp - j0;
        int32_t ng = 0;
        for (int64_t k0 = 0; k0 < vrows; k0 += kQrGramChunk, ++ng) {
          const float* vt = b.ptr<float>(s->Vt) + k0;
          float* g = b.ptr<float>(s->G) + size_t(ng) * kQrBlock * kQrBlock;
          gp.push_back(Prod{vt, vt, nullptr, g, s->dp, s->dp, 0, kQrBlock, kQrBlock, kQrBlock,
                            std::min<int64_t>(kQrGramChunk, vrows - k0), 1, 1.0f, 0.0f});
        }
        td.push_back(QrTDesc{b.ptr<float>(s->T), b.ptr<float>(s->G), ng});
      }
      add_wx(b, act, j0, kW, gp);
      add_gemm(b, gp);
      b.op(kOpQrT, td, int(td.size()));
    }
    // U = V T^T; X <- X - W U^T for the next block's columns first, then (on the auxiliary stream,
    // while the next block's panels run) for the rest of the trailing columns and for Q
    {
      std::vector<Prod> up;
      for (QrSide* s : act)
        up.push_back(Prod{b.ptr<float>(s->V), b.ptr<float>(s->T), nullptr, b.ptr<float>(s->U), kQrBlock, kQrBlock, 0,
                          kQrBlock, s->dp - j0, kQrBlock, kQrBlock, 0, 1.0f, 0.0f});
      add_gemm(b, up);
      std::vector<Prod> xn, xr;
      add_wx(b, act, j0, kXNext, xn);
      add_gemm(b, xn);
      add_wx(b, act, j0, kXRest, xr);
      b.fork();
      b.aux = 1;
      add_gemm(b, xr);
      b.aux = 0;
    }
  }
  b.join();
}

// Per matrix: left / right tell whether that side has a basis (its length is at most
// max_precond_dim); a side without one is the identity, and its statistic, basis buffers and
// product are skipped (kNone marks an unused buffer).
constexpr size_t kNone = ~size_t(0);
struct SoapPlan {
  int64_t m = 0, n = 0, mp = 0, np = 0;
  bool left = true, right = true;
  // the right product first: [G Q_R | M Q_R], then Q_L^T of it. Both orders take the same fp32
  // flop, but the product that reads a bf16 G takes three bf16 MFMAs per step instead of six, so
  // for a wide matrix (n > m) with a bf16 gradient and both bases the larger product is then the
  // cheaper one
  bool rfirst = false;
  // a side with a basis whose length is a multiple of the tile (and whose caller buffers are
  // 16-byte aligned, as the GEMM's vector accesses need) reads and updates the caller's statistic
  // where it lies and reads the caller's basis there (no copy in or out; the basis is still copied
  // transposed)
  bool lin = false, rin = false;
  size_t Gp = kNone, GMt = kNone, X1 = 0, GMr = 0, NpT = kNone, QLp = kNone, QLt = kNone, QRp = kNone,
         QRt = kNone, Lp = kNone, Rp = kNone;
  QrSide L, R;
};

constexpr int64_t kSoapMaxDim = 65536;  // sides without a basis

int64_t precond_limit(const mfsdp_soap_hparams* hp) { return hp->max_precond_dim == 0 ? kQrMaxDim : hp->max_precond_dim; }

int check_soap_hp(const mfsdp_soap_hparams* hp) {
  if (!hp) return bad("hparams is NULL");
  auto fin = [](double x) { return std::isfinite(x); };
  if (!(hp->lr >= 0.0) || !fin(hp->lr)) return bad("lr must be finite and >= 0");
  if (!(hp->weight_decay >= 0.0) || !fin(hp->weight_decay)) return bad("weight_decay must be finite and >= 0");
  if (!(hp->beta1 >= 0.0 && hp->beta1 < 1.0)) return bad("beta1 must be in [0, 1)");
  if (!(hp->beta2 >= 0.0 && hp->beta2 < 1.0)) return bad("beta2 must be in [0, 1)");
  if (!(hp->eps > 0.0) || !fin(hp->eps)) return bad("eps must be finite and > 0");
  if (!(hp->shampoo_beta >= 0.0) || !fin(hp->shampoo_beta)) return bad("shampoo_beta must be finite and >= 0");
  if (!(hp->shampoo_weight >= 0.0) || !fin(hp->shampoo_weight))
    return bad("shampoo_weight must be finite and >= 0");
  if (hp->step < 1) return bad("step must be >= 1");
  if (hp->refresh != 0 && hp->refresh != 1) return bad("refresh must be 0 or 1");
  if (hp->refresh_iters < 1 || hp->refresh_iters > 100) return bad("refresh_iters must be in [1, 100]");
  if (hp->max_precond_dim < 0 || hp->max_precond_dim > kQrMaxDim)
    return bad("max_precond_dim must be in [0, 4096] (0: 4096, the longest side a basis refresh supports)");
  return MFSDP_OK;
}

int check_soap_entries(const mfsdp_soap_entry* en, int64_t count, bool data, int64_t maxd) {
  if (count < 0) return bad("count must be >= 0");
  if (count > 0 && !en) return bad("entries is NULL");
  if (count > 4096) return bad("at most 4096 entries per call");
  int64_t units = 0;  // bound on the 64 x 64 tiles of any one grouped launch (grid and int32 counters)
  for (int64_t i = 0; i < count; ++i) {
    const mfsdp_soap_entry& e = en[i];
    const std::string w = "entry " + std::to_string(i) + ": ";
    if (e.m < 1 || e.n < 1 || e.m > kSoapMaxDim || e.n > kSoapMaxDim) return bad(w + "m and n must be in [1, 65536]");
    const int64_t s = rup(e.m, kShTile) + 2 * rup(e.n, kShTile);
    units += 3 * (s / kShCopyTile) * (s / kShCopyTile);
    if (units > (int64_t(1) << 30)) return bad("the entries of one call exceed 2^30 tiles per launch");
    if (!dtype_ok(e.param_dtype) || !dtype_ok(e.grad_dtype)) return bad(w + "dtype must be F32 or BF16");
    if (!data) continue;
    const bool left = e.m <= maxd, right = e.n <= maxd;
    if (!e.param || !e.grad || !e.exp_avg || !e.exp_avg_sq || (left && (!e.L || !e.QL)) || (right && (!e.R || !e.QR)))
      return bad(w + "NULL pointer");
    const size_t pa = e.param_dtype == MFSDP_BF16 ? 2 : 4, ga = e.grad_dtype == MFSDP_BF16 ? 2 : 4;
    if (!aligned(e.param, pa) || !aligned(e.grad, ga) || !aligned(e.exp_avg, 4) || !aligned(e.exp_avg_sq, 4) ||
        !aligned(e.L, 4) || !aligned(e.R, 4) || !aligned(e.QL, 4) || !aligned(e.QR, 4) ||
        !aligned(e.update_out, 4))
      return bad(w + "misaligned pointer");
  }
  return MFSDP_OK;
}

// `sizing`: for the size query, which sees no pointers (no side is then taken as in place: the
// most descriptors a step can need).
size_t build_soap(const mfsdp_soap_entry* en, int64_t count, const mfsdp_soap_hparams* hp, char* ws,
                  Build& b, size_t& desc_at, bool sizing) {
  b.base = ws;
  Arena a;
  const int64_t maxd = precond_limit(hp);
  std::vector<SoapPlan> P(static_cast<size_t>(count));
  for (int64_t i = 0; i < count; ++i) {
    SoapPlan& e = P[size_t(i)];
    e.m = en[i].m;
    e.n = en[i].n;
    e.left = e.m <= maxd;
    e.right = e.n <= maxd;
    e.mp = rup(e.m, kShTile);
    e.np = rup(e.n, kShTile);
    e.rfirst = e.left && e.right && e.n > e.m && en[i].grad_dtype == MFSDP_BF16;
    e.lin = !sizing && e.left && e.m == e.mp && aligned(en[i].L, 16) && aligned(en[i].QL, 16);
    e.rin = !sizing && e.right && e.n == e.np && aligned(en[i].R, 16) && aligned(en[i].QR, 16);
    const size_t f = sizeof(float), mn = size_t(e.mp) * size_t(e.np) * f;
    if (e.left) e.Gp = a.take(mn);               // G for the left statistic
    if (e.left || e.right) e.GMt = a.take(2 * mn);  // [G^T ; M^T]: left product, right statistic
    e.X1 = a.take(2 * mn);   // Q_L^T [G | M] (or [G | M] itself); later Z = Q_L N' (or N')
    e.GMr = a.take(2 * mn);  // [G' | M']; later N
    if (e.left) e.NpT = a.take(mn);
    if (e.left) {
      const size_t mm = size_t(e.mp) * size_t(e.mp) * f;
      e.QLp = a.take(mm);  // later the refresh product S^T = Q_L^T L
      e.QLt = a.take(mm);  // later the accumulated Q_L of the refresh
      e.Lp = a.take(mm);
      e.L.d = e.m;
      e.L.dp = e.mp;
      e.L.St = e.QLp;
      e.L.Q = e.QLt;
      plan_qr_buffers(e.L, a);
    }
    if (e.right) {
      const size_t nn = size_t(e.np) * size_t(e.np) * f;
      e.QRp = a.take(nn);
      e.QRt = a.take(nn);
      e.Rp = a.take(nn);
      e.R.d = e.n;
      e.R.dp = e.np;
      e.R.St = e.QRp;
      e.R.Q = e.QRt;
      plan_qr_buffers(e.R, a);
    }
  }
  desc_at = a.off;
  auto fp = [&](size_t off) { return off == kNone ? nullptr : b.ptr<float>(off); };
  // statistic and basis (row-major) of each side: the caller's buffers or their padded copies
  auto Lb = [&](const SoapPlan& e) { return e.lin ? en[&e - P.data()].L : b.ptr<float>(e.Lp); };
  auto Rb = [&](const SoapPlan& e) { return e.rin ? en[&e - P.data()].R : b.ptr<float>(e.Rp); };
  auto QLb = [&](const SoapPlan& e) { return e.lin ? en[&e - P.data()].QL : b.ptr<float>(e.QLp); };
  auto QRb = [&](const SoapPlan& e) { return e.rin ? en[&e - P.data()].QR : b.ptr<float>(e.QRp); };

  std::vector<ShCopyDesc> cin;
  std::vector<SoapPrepDesc> prep;
  int ct = 0, pt = 0;
  for (int64_t i = 0; i < count; ++i) {
    SoapPlan& e = P[size_t(i)];
    if (e.left) {
      if (!e.lin)
        cin.push_back(copy_desc(en[i].L, kDtF32, b.ptr<float>(e.Lp), nullptr, e.m, e.m, e.m, e.mp, 0, e.mp, e.mp, ct));
      cin.push_back(copy_desc(en[i].QL, kDtF32, e.lin ? nullptr : b.ptr<float>(e.QLp), b.ptr<float>(e.QLt), e.m, e.m,
                              e.m, e.mp, e.mp, e.mp, e.mp, ct));
    }
    if (e.right) {
      if (!e.rin)
        cin.push_back(copy_desc(en[i].R, kDtF32, b.ptr<float>(e.Rp), nullptr, e.n, e.n, e.n, e.np, 0, e.np, e.np, ct));
      cin.push_back(copy_desc(en[i].QR, kDtF32, e.rin ? nullptr : b.ptr<float>(e.QRp), b.ptr<float>(e.QRt), e.n, e.n,
                              e.n, e.np, e.np, e.np, e.np, ct));
    }
    SoapPrepDesc d{};
    d.grad = en[i].grad;
    d.exp_avg = en[i].exp_avg;
    d.Gp = fp(e.Gp);
    d.GMt = fp(e.GMt);
    d.GM = e.left ? nullptr : b.ptr<float>(e.X1);
    d.Mr = e.rfirst ? b.ptr<float>(e.GMt) + e.np * e.mp : nullptr;
    d.m = e.m;
    d.n = e.n;
    d.mp = e.mp;
    d.np = e.np;
    d.grad_dtype = en[i].grad_dtype == MFSDP_BF16 ? kDtBF16 : kDtF32;
    d.g_bf16 = d.grad_dtype == kDtBF16 ? 1 : 0;
    d.tiles_n = int32_t(e.np / kShCopyTile);
    d.tile_begin = pt;
    pt += int((e.mp / kShCopyTile) * (e.np / kShCopyTile));
    prep.push_back(d);
  }
  if (!cin.empty()) b.op(kOpCopyIn, cin, ct);
  b.op(kOpSoapPrep, prep, pt);

  // Products (a side without a basis skips its own):
  //   left:  X1 = Q_L^T [G | M];  Z = Q_L N' (from N'^T) into X1
  //   right: [G' | M'] = X1 halves Q_R into GMr;  N = Z Q_R^T into GMr
  //   (rfirst: X1 = Q_R^T [G^T | M^T], then [G' | M'] = Q_L^T X1^T into GMr; the rest as above)
  // Adam reads [G' | M'] from GMr (right) or X1 (no right basis) and writes N'^T (left) or N'
  // itself: into X1 as Z (right) or into GMr as N (neither); apply reads N from GMr, or from X1 when
  // only the left side has a basis.
  const float ws_ = float(hp->shampoo_weight), bs_ = float(hp->shampoo_beta);
  std::vector<Prod> p1, p2, p3, p4;
  for (SoapPlan& e : P) {
    float* X1 = b.ptr<float>(e.X1);
    float* GMr = b.ptr<float>(e.GMr);
    const int64_t mp = e.mp, np = e.np;
    // a bf16 gradient (stored as bf16 by the first-moment pass) is one bf16 part: one product per
    // statistic, three for Q_L^T G
    const bool gbf = en[&e - P.data()].grad_dtype == MFSDP_BF16;
    if (e.rfirst) {
      // X1 (as 2 np x mp, row stride mp) = [(G Q_R)^T ; (M Q_R)^T] = Q_R^T [G^T | M^T]; then
      // [G' | M'] = Q_L^T [G Q_R | M Q_R] into GMr; G is bf16 in Gp, M row-major after GMt's G^T rows
      const float* QRt = b.ptr<float>(e.QRt);
      const float* Mr = b.ptr<float>(e.GMt) + np * mp;
      p1.push_back(Prod{QRt, b.ptr<float>(e.Gp), nullptr, X1, np, np, 0, mp, np, mp, np, 0, 1.0f, 0.0f, false, true});
      p1.push_back(Prod{QRt, Mr, nullptr, X1 + np * mp, np, np, 0, mp, np, mp, np, 0, 1.0f, 0.0f});
      p2.push_back(Prod{b.ptr<float>(e.QLt), X1, nullptr, GMr, mp, mp, 0, 2 * np, mp, 2 * np, mp, 0, 1.0f, 0.0f});
    } else if (e.left) {
      const float* GMt = b.ptr<float>(e.GMt);
      // the G half of Q_L^T [G | M] has a one-part Q when the gradient is bf16
      p1.push_back(Prod{b.ptr<float>(e.QLt), GMt, nullptr, X1, mp, mp, 0, 2 * np, mp, np, mp, 0, 1.0f, 0.0f, false,
                        gbf});
      p1.push_back(Prod{b.ptr<float>(e.QLt), GMt + np * mp, nullptr, X1 + np, mp, mp, 0, 2 * np, mp, np, mp, 0,
                        1.0f, 0.0f});
    }
    if (e.left) {
      const float* Gp = b.ptr<float>(e.Gp);
      // the statistics read only G and G^T: they join the first launch
      p1.push_back(Prod{Gp, Gp, Lb(e), Lb(e), np, np, mp, mp, mp, mp, np, 1, ws_, bs_, gbf, gbf});
      p3.push_back(Prod{QLb(e), b.ptr<float>(e.NpT), nullptr, X1, mp, mp, 0, np, mp, np, mp, 0, 1.0f, 0.0f});
    }
    if (e.right) {
      const float* GMt = b.ptr<float>(e.GMt);
      p1.push_back(Prod{GMt, GMt, Rb(e), Rb(e), mp, mp, np, np, np, np, mp, 1, ws_, bs_, gbf, gbf});
      if (!e.rfirst)
        for (int h = 0; h < 2; ++h)
          p2.push_back(Prod{X1 + h * np, b.ptr<float>(e.QRt), nullptr, GMr + h * np, 2 * np, np, 0, 2 * np, mp, np,
                            np, 0, 1.0f, 0.0f});
      p4.push_back(Prod{X1, QRb(e), nullptr, GMr, np, np, 0, np, mp, np, np, 0, 1.0f, 0.0f});
    }
  }
  if (!p1.empty()) add_gemm(b, p1);
  if (!p2.empty()) add_gemm(b, p2);

  std::vector<SoapAdamDesc> ad;
  int at = 0;
  for (SoapPlan& e : P) {
    SoapAdamDesc d{};
    d.GMr = b.ptr<float>(e.right ? e.GMr : e.X1);
    d.exp_avg_sq = en[&e - P.data()].exp_avg_sq;
    d.NpT = fp(e.NpT);
    d.Np = e.left ? nullptr : b.ptr<float>(e.right ? e.X1 : e.GMr);
    d.m = e.m;
    d.n = e.n;
    d.mp = e.mp;
    d.np = e.np;
    d.tiles_n = int32_t(e.np / kShCopyTile);
    d.tile_begin = at;
    at += int((e.mp / kShCopyTile) * (e.np / kShCopyTile));
    ad.push_back(d);
  }
  b.op(kOpSoapAdam, ad, at);
  if (!p3.empty()) add_gemm(b, p3);
  if (!p4.empty()) add_gemm(b, p4);

  std::vector<ShApplyDesc> ap;
  int apt = 0;
  for (int64_t i = 0; i < count; ++i) {
    SoapPlan& e = P[size_t(i)];
    ShApplyDesc d{};
    d.U = b.ptr<float>((e.left && !e.right) ? e.X1 : e.GMr);
    d.ldu = e.np;
    d.param = en[i].param;
    d.update_out = en[i].update_out;
    d.m = e.m;
    d.n = e.n;
    d.param_dtype = en[i].param_dtype == MFSDP_BF16 ? kDtBF16 : kDtF32;
    const int64_t tn = (e.n + kShCopyTile - 1) / kShCopyTile, tm = (e.m + kShCopyTile - 1) / kShCopyTile;
    d.tiles_n = int32_t(tn);
    d.tile_begin = apt;
    apt += int(tm * tn);
    ap.push_back(d);
  }
  b.op(kOpApply, ap, apt);

  std::vector<ShCopyDesc> cst;
  ct = 0;
  for (int64_t i = 0; i < count; ++i) {
    SoapPlan& e = P[size_t(i)];
    if (e.left && !e.lin)
      cst.push_back(copy_desc(b.ptr<float>(e.Lp), kDtF32, en[i].L, nullptr, e.m, e.m, e.mp, e.m, 0, e.m, e.m, ct));
    if (e.right && !e.rin)
      cst.push_back(copy_desc(b.ptr<float>(e.Rp), kDtF32, en[i].R, nullptr, e.n, e.n, e.np, e.n, 0, e.n, e.n, ct));
  }
  if (!cst.empty()) b.op(kOpCopyOut, cst, ct);

  if (hp->refresh) {
    std::vector<Prod> ps;
    std::vector<QrSide*> sides;
    for (SoapPlan& e : P) {
      if (e.left) {
        ps.push_back(Prod{b.ptr<float>(e.QLt), Lb(e), nullptr, b.ptr<float>(e.QLp), e.mp, e.mp, 0, e.mp,
                          e.mp, e.mp, e.mp, 0, 1.0f, 0.0f});
        sides.push_back(&e.L);
      }
      if (e.right) {
        ps.push_back(Prod{b.ptr<float>(e.QRt), Rb(e), nullptr, b.ptr<float>(e.QRp), e.np, e.np, 0, e.np,
                          e.np, e.np, e.np, 0, 1.0f, 0.0f});
        sides.push_back(&e.R);
      }
    }
    if (!ps.empty()) {
      // one refresh = the power step S^T = basis^T statistic (S = statistic * basis), then the QR
      // of S, which leaves the new basis Q in the buffer that held the old basis transposed; a
      // further power step first transposes it back (a copy into the S^T buffer, then that buffer
      // copied onto itself with its transpose into the basis buffer). Repetitions reuse the first
      // one's descriptors.
      std::vector<ShCopyDesc> t1, t2;
      int n1 = 0, n2 = 0;
      for (QrSide* q : sides) {
        t1.push_back(copy_desc(b.ptr<float>(q->Q), kDtF32, b.ptr<float>(q->St), nullptr, q->d, q->d, q->dp, q->dp, 0,
                               q->dp, q->dp, n1));
        t2.push_back(copy_desc(b.ptr<float>(q->St), kDtF32, b.ptr<float>(q->St), b.ptr<float>(q->Q), q->d, q->d,
                               q->dp, q->dp, q->dp, q->dp, q->dp, n2));
      }
      const size_t first = b.ops.size();
      add_gemm(b, ps);
      add_qr_ops(b, sides);
      const size_t last = b.ops.size();
      for (int it = 1; it < hp->refresh_iters; ++it) {
        b.op(kOpCopyIn, t1, n1);
        b.op(kOpCopyIn, t2, n2);
        for (size_t k = first; k < last; ++k) {
          const Op o = b.ops[k];
          b.ops.push_back(o);
        }
      }
      std::vector<ShCopyDesc> co;
      int cot = 0;
      for (int64_t i = 0; i < count; ++i) {
        SoapPlan& e = P[size_t(i)];
        if (e.left)
          co.push_back(copy_desc(b.ptr<float>(e.QLt), kDtF32, en[i].QL, nullptr, e.m, e.m, e.mp, e.m, 0, e.m, e.m, cot));
        if (e.right)
          co.push_back(copy_desc(b.ptr<float>(e.QRt), kDtF32, en[i].QR, nullptr, e.n, e.n, e.np, e.n, 0, e.n, e.n, cot));
      }
      b.op(kOpCopyOut, co, cot);
    }
  }
  return desc_at + al(b.h.size());
}

size_t build_factor(int64_t d, const float* a, float* q, char* ws, Build& b, size_t& desc_at) {
  b.base = ws;
  Arena ar;
  QrSide s;
  s.d = d;
  s.dp = rup(d, kShTile);
  const size_t mat = size_t(s.dp) * size_t(s.dp) * sizeof(float);
  s.St = ar.take(mat);
  s.Q = ar.take(mat);
  plan_qr_buffers(s, ar);
  desc_at = ar.off;
  std::vector<ShCopyDesc> cin;
  int ct = 0;
  // St = a^T (the Q buffer takes a itself, then the identity)
  cin.push_back(copy_desc(a, kDtF32, b.ptr<float>(s.Q), b.ptr<float>(s.St), d, d, d, s.dp, s.dp, s.dp, s.dp, ct));
  b.op(kOpCopyIn, cin, ct);
  std::vector<QrSide*> sides{&s};
  add_qr_ops(b, sides);
  std::vector<ShCopyDesc> co;
  int cot = 0;
  co.push_back(copy_desc(b.ptr<float>(s.Q), kDtF32, q, nullptr, d, d, s.dp, d, 0, d, d, cot));
  b.op(kOpCopyOut, co, cot);
  return desc_at + al(b.h.size());
}

int workspace_error(size_t need, const char* query) {
  return set_last_error(MFSDP_E_WORKSPACE, std::string("workspace NULL, not 256-byte aligned or smaller than ") +
                                               query + " (" + std::to_string(need) + " bytes)");
}

}  // namespace

extern "C" {

size_t mfsdp_soap_workspace_size(const mfsdp_soap_entry* entries, int64_t count, const mfsdp_soap_hparams* hp) {
  if (check_soap_hp(hp) != MFSDP_OK) return 0;
  if (check_soap_entries(entries, count, false, precond_limit(hp)) != MFSDP_OK) return 0;
  if (count == 0) return 0;
  Build b;
  size_t desc_at = 0;
  return build_soap(entries, count, hp, nullptr, b, desc_at, true);
}

int mfsdp_soap_step(const mfsdp_soap_entry* entries, int64_t count, const mfsdp_soap_hparams* hp,
                    void* workspace, size_t workspace_bytes, void* stream) {
  int rc = check_soap_hp(hp);
  if (rc != MFSDP_OK) return rc;
  rc = check_soap_entries(entries, count, true, precond_limit(hp));
  if (rc != MFSDP_OK) return rc;
  if (count == 0) return MFSDP_OK;
  Build b;
  size_t desc_at = 0;
  const size_t need = build_soap(entries, count, hp, static_cast<char*>(workspace), b, desc_at, false);
  if (!workspace || !aligned(workspace, kAl) || workspace_bytes < need)
    return workspace_error(need, "mfsdp_soap_workspace_size");
  RunScalars rs;
  rs.decay = float(1.0 - hp->lr * hp->weight_decay);
  rs.step = float(hp->lr);
  rs.beta1 = float(hp->beta1);
  rs.beta2 = float(hp->beta2);
  rs.adam_eps = float(hp->eps);
  rs.inv_bc1 = float(1.0 / (1.0 - std::pow(hp->beta1, double(hp->step))));
  rs.inv_sqrt_bc2 = float(1.0 / std::sqrt(1.0 - std::pow(hp->beta2, double(hp->step))));
  return run(b, static_cast<char*>(workspace), desc_at, static_cast<hipStream_t>(stream), rs);
}

size_t mfsdp_orthonormal_factor_workspace_size(int64_t d) {
  if (d < 1 || d > kQrMaxDim) return 0;
  Build b;
  size_t desc_at = 0;
  return build_factor(d, nullptr, nullptr, nullptr, b, desc_at);
}

int mfsdp_orthonormal_factor(const float* a, float* q, int64_t d, void* workspace, size_t workspace_bytes,
                             void* stream) {
  if (!a || !q) return bad("a and q must be non-NULL");
  if (!aligned(a, 4) || !aligned(q, 4)) return bad("misaligned pointer");
  if (d < 1 || d > kQrMaxDim) return bad("d must be in [1, 4096]");
  Build b;
  size_t desc_at = 0;
  const size_t need = build_factor(d, a, q, static_cast<char*>(workspace), b, desc_at);
  if (!workspace || !aligned(workspace, kAl) || workspace_bytes < need)
    return workspace_error(need, "mfsdp_orthonormal_factor_workspace_size");
  return run(b, static_cast<char*>(workspace), desc_at, static_cast<hipStream_t>(stream), RunScalars{});
}

}  // extern "C"
