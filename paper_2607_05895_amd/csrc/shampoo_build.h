// Launch-sequence builder shared by the Shampoo-family host code (Shampoo, the inverse root, SOAP,
// the orthonormal factor): a workspace bump allocator, descriptor arrays packed in one host buffer
// (uploaded once into the workspace through the pinned staging ring) and the ops that consume them,
// all enqueued on the caller's stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstring>
#include <string>
#include <vector>

#include "../../include/mfsdp.h"
#include "mfsdp_internal.h"
#include "shampoo_internal.h"
#include "soap_internal.h"

namespace mfsdp {
int set_last_error(int status, const std::string& msg);
int staging_acquire(size_t bytes, void** host);
int staging_upload(int slot, void* dst, size_t bytes, hipStream_t st);
// The device's auxiliary stream and (if ev is set) the next event of its ring.
int aux_stream(hipStream_t* out, hipEvent_t* ev);

namespace shb {

constexpr size_t kAl = 256;
inline size_t al(size_t x) { return (x + kAl - 1) / kAl * kAl; }
inline int64_t rup(int64_t x, int64_t a) { return (x + a - 1) / a * a; }
inline int bad(const std::string& m) { return set_last_error(MFSDP_E_INVALID, m); }
inline int hip_err(hipError_t e, const char* what) {
  return set_last_error(MFSDP_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}
inline bool dtype_ok(int32_t dt) { return dt == MFSDP_F32 || dt == MFSDP_BF16; }
inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Workspace bump allocator (offsets only; the base is added when the workspace is known).
struct Arena {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off = al(off + bytes);
    return o;
  }
};

enum OpKind {
  kOpCopyIn, kOpCopyOut, kOpGemm, kOpNorm, kOpScalars, kOpInit, kOpApply,
  kOpSoapPrep, kOpSoapAdam, kOpEye, kOpQrPanel, kOpQrCol, kOpQrT,
  kOpFork,  // the auxiliary stream waits for everything enqueued so far on the caller's stream
  kOpJoin   // the caller's stream waits for everything enqueued so far on the auxiliary stream
};
struct Op {
  OpKind kind;
  size_t desc_off;
  int count;
  int total;  // grid blocks
  int aux;    // 1: launched on the auxiliary stream
};

// Per-call scalars the kernels take by value.
struct RunScalars {
  double eps = 0.0, eps_rel = 0.0;  // inverse-root ridge
  int p = 4;                        // inverse-root order
  float decay = 1.0f, step = 0.0f;  // parameter update p <- p decay - step U
  float beta1 = 0.0f, beta2 = 0.0f, adam_eps = 0.0f, inv_bc1 = 1.0f, inv_sqrt_bc2 = 1.0f;  // SOAP
};

struct Build {
  char* base = nullptr;  // workspace base (nullptr while sizing)
  std::vector<char> h;
  std::vector<Op> ops;
  template <class T>
  T* ptr(size_t off) const {  // integer arithmetic: base is null while only sizing
    return reinterpret_cast<T*>(reinterpret_cast<uintptr_t>(base) + off);
  }
  template <class T>
  size_t put(const std::vector<T>& v) {
    const size_t o = al(h.size());
    h.resize(o + v.size() * sizeof(T));
    std::memcpy(h.data() + o, v.data(), v.size() * sizeof(T));
    return o;
  }
  int aux = 0;  // stream of the ops added next
  template <class T>
  void op(OpKind k, const std::vector<T>& v, int total) {
    if (v.empty() || total <= 0) return;
    ops.push_back(Op{k, put(v), int(v.size()), total, aux});
  }
  void fork() { ops.push_back(Op{kOpFork, 0, 0, 0, 0}); }
  void join() { ops.push_back(Op{kOpJoin, 0, 0, 0, 0}); }
};

inline ShCopyDesc copy_desc(const void* src, int dt, void* dst, void* dstT, int64_t rows, int64_t cols,
                            int64_t ld_src, int64_t ld_dst, int64_t ld_dstT, int64_t dom_rows,
                            int64_t dom_cols, int& tiles) {
  ShCopyDesc c{};
  c.src = src;
  c.dst = dst;
  c.dstT = dstT;
  c.rows = rows;
  c.cols = cols;
  c.ld_src = ld_src;
  c.ld_dst = ld_dst;
  c.ld_dstT = ld_dstT;
  c.src_dtype = dt;
  const int64_t tm = (dom_rows + kShCopyTile - 1) / kShCopyTile;
  const int64_t tn = (dom_cols + kShCopyTile - 1) / kShCopyTile;
  c.tiles_n = int32_t(tn);
  c.tile_begin = tiles;
  tiles += int(tm * tn);
  return c;
}

inline ShGemmDesc gemm_desc(const float* P, const float* Q, const float* E, float* C, int64_t ldp,
                            int64_t ldq, int64_t lde, int64_t ldc, int64_t M, int64_t N, int64_t K,
                            int sym, float alpha, float beta, float diag, int& tiles) {
  ShGemmDesc g{};
  g.P = P;
  g.Q = Q;
  g.E = E;
  g.C = C;
  g.ldp = ldp;
  g.ldq = ldq;
  g.lde = lde;
  g.ldc = ldc;
  g.K = int32_t(K);
  g.tiles_n = int32_t(N / kShTile);
  g.sym = sym;
  g.alpha = alpha;
  g.beta = beta;
  g.diag = diag;
  g.tile_begin = tiles;
  const int64_t tm = M / kShTile, tn = N / kShTile;
  tiles += int(sym ? tn * (tn + 1) / 2 : tm * tn);
  return g;
}

inline int run(Build& b, char* ws, size_t desc_at, hipStream_t main_st, const RunScalars& s) {
  hipStream_t st = main_st;
  if (!b.h.empty()) {
    void* host = nullptr;
    const int slot = staging_acquire(b.h.size(), &host);
    if (slot < 0) return slot;
    std::memcpy(host, b.h.data(), b.h.size());
    const int rc = staging_upload(slot, ws + desc_at, b.h.size(), st);
    if (rc != MFSDP_OK) return rc;
  }
  hipStream_t aux = nullptr;
  bool forked = false;
  for (const Op& o : b.ops) {
    if (o.kind == kOpFork || o.kind == kOpJoin) {
      hipEvent_t ev = nullptr;
      const int rc = aux_stream(&aux, &ev);
      if (rc != MFSDP_OK) return rc;
      hipError_t e = hipEventRecord(ev, o.kind == kOpFork ? main_st : aux);
      if (e == hipSuccess) e = hipStreamWaitEvent(o.kind == kOpFork ? aux : main_st, ev, 0);
      if (e != hipSuccess) return hip_err(e, "stream fork / join");
      forked = o.kind == kOpFork;
      continue;
    }
    char* dp = ws + desc_at + o.desc_off;
    hipError_t e = hipSuccess;
    if (o.aux && !forked) return set_last_error(MFSDP_E_INVALID, "internal: auxiliary-stream op outside a fork");
    st = o.aux ? aux : main_st;
    switch (o.kind) {
      case kOpCopyIn: e = launch_sh_copy(reinterpret_cast<ShCopyDesc*>(dp), o.count, o.total, 0, st); break;
      case kOpCopyOut: e = launch_sh_copy(reinterpret_cast<ShCopyDesc*>(dp), o.count, o.total, 1, st); break;
      case kOpGemm: e = launch_sh_gemm(reinterpret_cast<ShGemmDesc*>(dp), o.count, o.total, st); break;
      case kOpNorm: e = launch_sh_norm(reinterpret_cast<ShNormDesc*>(dp), o.count, o.total, st); break;
      case kOpScalars:
        e = launch_sh_scalars(reinterpret_cast<ShScalarDesc*>(dp), o.count, s.eps, s.eps_rel, s.p, st);
        break;
      case kOpInit: e = launch_sh_init(reinterpret_cast<ShInitDesc*>(dp), o.count, o.total, st); break;
      case kOpApply:
        e = launch_sh_apply(reinterpret_cast<ShApplyDesc*>(dp), o.count, o.total, s.decay, s.step, st);
        break;
      case kOpSoapPrep:
        e = launch_soap_prep(reinterpret_cast<SoapPrepDesc*>(dp), o.count, o.total, s.beta1, st);
        break;
      case kOpSoapAdam:
        e = launch_soap_adam(reinterpret_cast<SoapAdamDesc*>(dp), o.count, o.total, s.beta2, s.adam_eps,
                             s.inv_bc1, s.inv_sqrt_bc2, st);
        break;
      case kOpEye: e = launch_soap_eye(reinterpret_cast<SoapEyeDesc*>(dp), o.count, o.total, st); break;
      case kOpQrPanel: e = launch_qr_panel(reinterpret_cast<QrPanelDesc*>(dp), o.count, st); break;
      case kOpQrCol: e = launch_qr_col(reinterpret_cast<QrColDesc*>(dp), o.count, o.total, st); break;
      case kOpQrT: e = launch_qr_t(reinterpret_cast<QrTDesc*>(dp), o.count, st); break;
      case kOpFork:
      case kOpJoin:
        break;
    }
    if (e != hipSuccess) return hip_err(e, "kernel launch");
  }
  if (forked) return set_last_error(MFSDP_E_INVALID, "internal: auxiliary stream not joined");
  return MFSDP_OK;
}

}  // namespace shb
}  // namespace mfsdp
