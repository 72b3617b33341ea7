/*
 * mfsdp.h -- C ABI of the owner-local Muon / AdamW step for MI355X (gfx950).
 *
 * MatrixFSDP (arxiv 2607.05895) places every data-parallel-sharded 2D weight whole on one owner
 * rank. After backward the owner holds the complete gradient of each matrix it owns and runs the
 * Muon update on it locally, with no collective (Section 3; Section 4.4 routes each owned full
 * matrix to Muon and the packed non-matrix "tail" tensors to AdamW). This library is that
 * owner-side computation on one GPU:
 *
 *   mfsdp_muon_step      -- Muon over a heterogeneous list of whole matrices the rank owns
 *   mfsdp_newton_schulz  -- the Newton-Schulz orthogonalisation of one matrix
 *   mfsdp_adamw_step     -- AdamW over the rank's tail tensors
 *
 * Muon, per owned matrix with stored shape m x n (Section 5.1 uses torch.optim.Muon's update):
 *   buf <- buf + (1 - beta) (g - buf)                    momentum EMA
 *   u   <- g + beta (buf - g)   (Nesterov) or  u <- buf
 *   X   <- u, or u^T when m > n  (r = min(m,n) rows, s = max(m,n) columns)
 *   X   <- X / max(||X||_F, eps)
 *   K times:  A = X X^T;  B = b A + c A A;  X <- a X + B X      (quintic NS)
 *   O   <- X, transposed back when m > n
 *   p   <- p (1 - lr wd) - lr f(m, n) O
 *   f = 1 | sqrt(max(1, m/n)) | 0.2 sqrt(max(m, n))   (lr_adjust NONE | ORIGINAL | MATCH_RMS_ADAMW)
 *
 * Conventions shared by every entry point
 *   - Pointers are device pointers (hipMalloc'd memory, e.g. torch CUDA tensors), contiguous
 *     row-major, 16-byte aligned. The caller owns every buffer: parameters, gradients, optimizer
 *     state, workspace and optional outputs. The library never frees or keeps them.
 *   - Calls are asynchronous: they validate, enqueue kernels on `stream` (a hipStream_t, NULL =
 *     the null stream) and return. Buffers must stay alive until the stream work completes.
 *     A workspace may be reused by the next call on the same stream; calls on different streams
 *     need different workspaces.
 *   - Every argument check runs before anything is enqueued: on error nothing is modified.
 *   - Results are deterministic: identical inputs give bitwise-identical outputs (fixed reduction
 *     orders, no floating-point atomics).
 *   - Non-finite inputs propagate; they are not checked.
 *   - Entries must not overlap each other; grad must not alias param or state. Not checked.
 *   - Return 0 on success, a negative mfsdp_status on failure; mfsdp_last_error() then describes
 *     the failure (thread-local text).
 */
#ifndef MFSDP_H
#define MFSDP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MFSDP_ABI_VERSION 6

typedef enum { MFSDP_F32 = 0, MFSDP_BF16 = 1 } mfsdp_dtype;

typedef enum {
  MFSDP_LR_NONE = 0,            /* f = 1 */
  MFSDP_LR_ORIGINAL = 1,        /* f = sqrt(max(1, m/n))  (torch.optim.Muon default) */
  MFSDP_LR_MATCH_RMS_ADAMW = 2  /* f = 0.2 sqrt(max(m, n))  (the paper's setting, Section 5.1) */
} mfsdp_lr_adjust;

typedef enum {
  MFSDP_OK = 0,
  MFSDP_E_INVALID = -1,    /* bad argument: NULL, size <= 0, dtype, alignment, hyperparameter */
  MFSDP_E_WORKSPACE = -2,  /* workspace NULL, misaligned or smaller than the size query */
  MFSDP_E_HIP = -3         /* a HIP runtime call or kernel launch failed */
} mfsdp_status;

/* One whole matrix the rank owns (Section 3: the owner's full 2D shard).
 *   param      m x n, param_dtype (F32 or BF16), updated in place (fp32 math, bf16 stored with
 *              round-to-nearest-even)
 *   grad       m x n, grad_dtype (F32 or BF16), read only
 *   momentum   m x n fp32 Muon buffer, updated in place
 *   m, n       stored rows and columns (the parameter's shape), both >= 1
 *   update_out optional m x n fp32: receives O (the NS output, before lr scaling). NULL = off. */
typedef struct {
  void* param;
  const void* grad;
  float* momentum;
  int64_t m;
  int64_t n;
  int32_t param_dtype;
  int32_t grad_dtype;
  float* update_out;
} mfsdp_muon_entry;

/* Muon hyperparameters, shared by every entry of one call. Given in double precision; derived
 * constants (1 - momentum, 1 - lr wd, lr f) are formed in double and rounded once to fp32.
 *   lr >= 0, weight_decay >= 0, 0 <= momentum < 1, nesterov 0/1,
 *   (a, b, c) NS coefficients, 0 <= ns_steps < 100, eps > 0 (norm clamp),
 *   lr_adjust an mfsdp_lr_adjust, ns_dtype: BF16 = NS products on bf16 MFMA with fp32
 *   accumulation and bf16 storage between products; F32 = fp32 throughout.
 *   ns_schedule: NULL = the triple (a, b, c) on every NS step; otherwise a host array of ns_steps
 *   finite triples (a_k, b_k, c_k), k = 0 .. ns_steps - 1, step k computing
 *   X <- a_k X + (b_k A + c_k A A) X. It is read during the call and not kept. (The paper runs one
 *   fixed triple; a constant schedule is identical to it.) */
typedef struct {
  double lr;
  double weight_decay;
  double momentum;
  int32_t nesterov;
  double a, b, c;
  int32_t ns_steps;
  double eps;
  int32_t lr_adjust;
  int32_t ns_dtype;
  const double* ns_schedule;
} mfsdp_muon_hparams;

/* One tail tensor (Section 4.4: non-matrix tensors stay on AdamW), flattened.
 *   param, grad  numel elements of param_dtype / grad_dtype (F32 or BF16)
 *   exp_avg, exp_avg_sq  numel fp32 moments, updated in place. */
typedef struct {
  void* param;
  const void* grad;
  float* exp_avg;
  float* exp_avg_sq;
  int64_t numel;
  int32_t param_dtype;
  int32_t grad_dtype;
} mfsdp_adamw_entry;

/* Bytes of device workspace mfsdp_muon_step (and mfsdp_muon_step_reduce) needs for these entries
 * and hyperparameters (Newton-Schulz iterates in both layouts, the r x r Gram and polynomial
 * matrices, norm partials, launch descriptors and, when the Gram product of a call has fewer tiles
 * than the GPU has compute units and some of its contractions are long, fp32 partial tiles of
 * those contractions split into ranges: at most a quarter of the rest); the entries' data
 * pointers are not used.
 * Returns 0 if the arguments are invalid (see mfsdp_last_error). count == 0 returns 0 with no
 * error. */
size_t mfsdp_muon_workspace_size(const mfsdp_muon_entry* entries, int64_t count,
                                 const mfsdp_muon_hparams* hp);

/* The owner's Muon step (Section 3; hyperparameters as in Section 5.1) for every entry.
 * workspace: device memory of at least mfsdp_muon_workspace_size bytes, 256-byte aligned; its
 * contents on entry are ignored and on return are unspecified. count == 0 is a no-op. */
int mfsdp_muon_step(const mfsdp_muon_entry* entries, int64_t count, const mfsdp_muon_hparams* hp,
                    void* workspace, size_t workspace_bytes, void* stream);

/* mfsdp_muon_step that also records caller-created HIP events (hipEvent_t, any may be NULL) on
 * `stream` at the phase boundaries of the step, for timing each phase on the stream it runs on:
 *   events[0] before the momentum pass, events[1] before the first Newton-Schulz product,
 *   events[2] after the last Newton-Schulz product, events[3] after the parameter update.
 * `events` itself may be NULL (then identical to mfsdp_muon_step). */
int mfsdp_muon_step_timed(const mfsdp_muon_entry* entries, int64_t count,
                          const mfsdp_muon_hparams* hp, void* workspace, size_t workspace_bytes,
                          void* stream, void* const* events);

/* Size of the static device array mfsdp_muon_step_noalloc works in: 64 MiB per GPU the library runs
 * on, held until the process ends. It fits, e.g., one 2048 x 2048 or one 1024 x 4096 matrix, or eight
 * 768 x 768 matrices (mfsdp_muon_workspace_size gives what a list of entries needs). */
#define MFSDP_NOALLOC_SCRATCH_BYTES (64u << 20)

/* mfsdp_muon_step for callers that cannot allocate memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation. Same entries, hyperparameters, results (bitwise
 * those of mfsdp_muon_step) and error rules, but no workspace argument and no allocation of any kind
 * by the library (no hipMalloc / hipFree / hipHostMalloc; the launch descriptors are passed to the
 * device as kernel arguments, a few small launches per call, instead of through pinned staging).
 *   - The workspace is a file-scope device array of MFSDP_NOALLOC_SCRATCH_BYTES, one per GPU. Entries
 *     whose mfsdp_muon_workspace_size exceeds it are rejected with MFSDP_E_INVALID before anything is
 *     enqueued; use mfsdp_muon_step with a caller workspace for them.
 *   - The call runs on the current device; `stream` (hipStream_t, NULL = null stream) must belong to
 *     it. The first call on a device looks up that device's copy of the array (hipGetSymbolAddress);
 *     make one call before capturing a graph so that the lookup is not part of the capture.
 *   - Every call on one GPU shares that GPU's array, which keeps the last call's contents (nothing in
 *     it needs to start at zero: each call writes every byte it reads). Calls that overlap on one
 *     GPU (different streams, threads, or graph replays running concurrently) race on it and give
 *     wrong results: order them on one stream or with events. */
int mfsdp_muon_step_noalloc(const mfsdp_muon_entry* entries, int64_t count,
                            const mfsdp_muon_hparams* hp, void* stream);

/* Most gradient parts one entry of mfsdp_muon_step_reduce may have (the paper's largest shard
 * span is 64 ranks). */
#define MFSDP_MAX_GRAD_PARTS 64

/* Owner-side gradient reduction fused with the Muon step. In owner placement every rank of the
 * shard span contributes its full-gradient buffer of a matrix and the reduced result is kept only
 * in the owner's segment (Section 4.2, owner-segment collectives); here the owner has received the
 * nparts contributions and the reduction runs inside the momentum pass. For entry i the Muon input
 * gradient is
 *     g_i = grad_scale * (P_i0 + P_i1 + ... + P_i,nparts-1)      (fp32, summed in that order)
 * with P_iw = grad_parts[i * nparts + w]: m x n, entries[i].grad_dtype, device memory, read only,
 * 16-byte aligned. grad_scale = 1 / nparts gives the data-parallel mean; it must be finite.
 *   1 <= nparts <= MFSDP_MAX_GRAD_PARTS; entries[i].grad is not read (may be NULL).
 *   reduced_out: NULL, or a host array of count device pointers, each NULL or an m x n buffer of
 *                grad_dtype (16-byte aligned) that receives g_i (bf16: round to nearest even).
 * Everything else as mfsdp_muon_step (same workspace size query); g_i enters the momentum pass
 * unrounded. */
int mfsdp_muon_step_reduce(const mfsdp_muon_entry* entries, int64_t count,
                           const void* const* grad_parts, int32_t nparts, double grad_scale,
                           void* const* reduced_out, const mfsdp_muon_hparams* hp, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Bytes of workspace mfsdp_newton_schulz needs for one m x n matrix. 0 on invalid input. */
size_t mfsdp_ns_workspace_size(int64_t m, int64_t n, int32_t ns_dtype);

/* out = NS_steps(x / max(||x||_F, eps)) for one m x n matrix (Section 2: iterations of
 * whole-matrix products X X^T), transposing internally when m > n.
 *   x    m x n, x_dtype (F32 or BF16), read only
 *   out  m x n, out_dtype (F32 or BF16); must not alias x
 *   ns_dtype as in mfsdp_muon_hparams; workspace sized by mfsdp_ns_workspace_size. */
int mfsdp_newton_schulz(const void* x, int32_t x_dtype, void* out, int32_t out_dtype, int64_t m,
                        int64_t n, double a, double b, double c, int32_t steps, double eps,
                        int32_t ns_dtype, void* workspace, size_t workspace_bytes, void* stream);

/* mfsdp_newton_schulz with one coefficient triple per step: coeffs is a host array of `steps`
 * finite triples (a_k, b_k, c_k) (read during the call, not kept); NULL is invalid unless
 * steps == 0. Same workspace size. */
int mfsdp_newton_schulz_schedule(const void* x, int32_t x_dtype, void* out, int32_t out_dtype,
                                 int64_t m, int64_t n, const double* coeffs, int32_t steps,
                                 double eps, int32_t ns_dtype, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* AdamW on the tail tensors (Section 4.4; PyTorch AdamW per Section 5.1):
 *   p <- p (1 - lr wd);  m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2
 *   p <- p - lr / (1 - beta1^t) * m / (sqrt(v) / sqrt(1 - beta2^t) + eps)
 * step = t >= 1 is the step number after increment. lr, wd >= 0; betas in [0, 1); eps > 0.
 * Hyperparameters are doubles; 1 - beta, the bias corrections and lr / (1 - beta1^t) are formed in
 * double and rounded once to fp32 (the elementwise math is fp32).
 * Needs no workspace. count == 0 is a no-op. */
int mfsdp_adamw_step(const mfsdp_adamw_entry* entries, int64_t count, double lr, double beta1,
                     double beta2, double eps, double weight_decay, int64_t step, void* stream);

/* ---- Shampoo owner step (Section 5.7: a single-device matrix optimizer on the owner) --------- */

/* One whole matrix the rank owns, for Shampoo (Gupta, Koren and Singer 2018, the matrix case:
 * full left and right preconditioners with the inverse fourth root, as the paper runs it).
 *   param      m x n, param_dtype (F32 or BF16), updated in place (fp32 math, bf16 rounded to
 *              nearest even)
 *   grad       m x n, grad_dtype (F32 or BF16), read only
 *   L, R       m x m and n x n fp32 statistics (row-major), updated in place; start at zero
 *   PL, PR     m x m and n x n fp32 preconditioners (row-major): written when hp->refresh is 1,
 *              read (and left unchanged) when it is 0
 *   m, n       1 .. 65536
 *   update_out optional m x n fp32: receives U = PL G PR. NULL = off.
 * All buffers are distinct device allocations (no aliasing), naturally aligned. */
typedef struct {
  void* param;
  const void* grad;
  float* L;
  float* R;
  float* PL;
  float* PR;
  int64_t m;
  int64_t n;
  int32_t param_dtype;
  int32_t grad_dtype;
  float* update_out;
} mfsdp_shampoo_entry;

/* Shampoo hyperparameters, shared by every entry of one call (doubles; fp32 math on the GPU).
 *   lr >= 0, weight_decay >= 0: p <- p (1 - lr wd) - lr U (decoupled decay, both on the old p)
 *   beta >= 0, weight >= 0: S <- beta S + weight G G^T (L) and G^T G (R); 1, 1 = accumulation
 *   eps > 0, eps_rel >= 0: the root is taken of S + rho I, rho = eps + eps_rel ||S||_F
 *   refresh 0/1: recompute PL, PR from the updated statistics (1) or use the stored ones (0)
 *   root_iters 1 .. 100: iterations of the coupled Newton inverse-root iteration (20 reaches fp32
 *   accuracy for rho >= 1e-6 ||S||_F on the tested spectra; see mfsdp_inverse_root). */
typedef struct {
  double lr;
  double weight_decay;
  double beta;
  double weight;
  double eps;
  double eps_rel;
  int32_t refresh;
  int32_t root_iters;
} mfsdp_shampoo_hparams;

/* Bytes of device workspace mfsdp_shampoo_step needs for these entries and hyperparameters:
 * per matrix, zero-padded copies of G and G^T (fp32, or bf16 for a bf16 gradient), P_L G and U
 * (3 mp np floats in all) and five
 * padded matrices per side for the root iteration (5 (mp^2 + np^2) floats), mp, np = m, n rounded
 * up to 128; plus launch descriptors. Data pointers are not used. 0 on invalid arguments;
 * count == 0 returns 0 with no error. */
size_t mfsdp_shampoo_workspace_size(const mfsdp_shampoo_entry* entries, int64_t count,
                                    const mfsdp_shampoo_hparams* hp);

/* One Shampoo step on every entry (host array of count entries), enqueued on `stream`
 * (hipStream_t, NULL = default stream); no host synchronisation. Statistics update, inverse
 * fourth roots (on refresh), U = P_L G P_R, every product at fp32 accuracy on the bf16 MFMA
 * (each fp32 operand split exactly into three bf16 parts, fp32 accumulation), then the parameter
 * update. The workspace (device, 256-byte aligned, >= the size query) must not be in use by
 * another call still running. Returns MFSDP_OK, MFSDP_E_INVALID, MFSDP_E_WORKSPACE or
 * MFSDP_E_HIP; on an argument error nothing is enqueued. At most 4096 entries per call. */
int mfsdp_shampoo_step(const mfsdp_shampoo_entry* entries, int64_t count,
                       const mfsdp_shampoo_hparams* hp, void* workspace, size_t workspace_bytes,
                       void* stream);

/* Workspace bytes for mfsdp_inverse_root (0 on invalid arguments). */
size_t mfsdp_inverse_root_workspace_size(int64_t d, int32_t p, int32_t iters);

/* out = (a + rho I)^(-1/p), rho = eps + eps_rel ||a||_F, for a symmetric positive semidefinite
 * d x d fp32 matrix `a` (row-major, device; read only; not checked for symmetry), by `iters`
 * steps of the coupled Newton iteration (Guo and Higham 2006), the iteration the Shampoo step
 * uses (products as there). p in {1, 2, 4}; 1 <= d <= 65536; eps > 0; eps_rel >= 0;
 * 1 <= iters <= 100.
 * `out` (d x d fp32, device) must not overlap `a`. In fp32 the iteration is stable while rho is
 * at least about 1e-6 ||a||_F; a smaller ridge can diverge. Same stream, workspace and error
 * rules as mfsdp_shampoo_step. */
int mfsdp_inverse_root(const float* a, float* out, int64_t d, int32_t p, double eps,
                       double eps_rel, int32_t iters, void* workspace, size_t workspace_bytes,
                       void* stream);

/* ---- SOAP owner step (Section 5.7: Adam in the eigenbasis of Shampoo's statistics) ---------- */

/* One whole matrix the rank owns, for SOAP (Vyas et al. 2024, the matrix case). A side longer than
 * the call's max_precond_dim (hparams) has no basis: it is the identity, that side's statistic is
 * not kept, and its L (or R) and QL (or QR) are not read or written (they may be NULL).
 *   param       m x n, param_dtype (F32 or BF16), updated in place (fp32 math, bf16 rounded to
 *               nearest even)
 *   grad        m x n, grad_dtype (F32 or BF16), read only
 *   exp_avg     m x n fp32 first moment M in the original coordinates, updated in place
 *   exp_avg_sq  m x n fp32 second moment V in the eigenbasis coordinates, updated in place
 *   L, R        m x m and n x n fp32 Shampoo statistics (row-major), updated in place
 *   QL, QR      m x m and n x n fp32 orthogonal bases (row-major; columns are the basis vectors):
 *               read; overwritten by the refreshed bases when hp->refresh is 1. Start them at the
 *               identity (then the first steps are AdamW steps).
 *   m, n        1 .. 65536; a side with a basis is at most max_precond_dim <= 4096 long (its basis
 *               is refreshed by a QR whose panels are held in registers, at most 4096 rows)
 *   update_out  optional m x n fp32: receives the direction N. NULL = off.
 * All buffers are distinct device allocations (no aliasing), naturally aligned. */
typedef struct {
  void* param;
  const void* grad;
  float* exp_avg;
  float* exp_avg_sq;
  float* L;
  float* R;
  float* QL;
  float* QR;
  int64_t m;
  int64_t n;
  int32_t param_dtype;
  int32_t grad_dtype;
  float* update_out;
} mfsdp_soap_entry;

/* SOAP hyperparameters, shared by every entry of one call (doubles; fp32 math on the GPU). Per
 * step, with the bases of the previous refresh:
 *   G' = QL^T G QR;  M <- beta1 M + (1 - beta1) G;  M' = QL^T M QR;  V <- beta2 V + (1 - beta2) G'^2
 *   N' = (M' / (1 - beta1^t)) / (sqrt(V) / sqrt(1 - beta2^t) + eps);  N = QL N' QR^T
 *   p <- p (1 - lr wd) - lr N      (decoupled decay, both terms on the old p)
 *   L <- shampoo_beta L + shampoo_weight G G^T;  R <- shampoo_beta R + shampoo_weight G^T G
 *   refresh 1: refresh_iters times QL <- Q factor of the Householder QR of L QL (and R, QR alike),
 *   with LAPACK's sign convention; refresh 0: the bases are read only.
 *   max_precond_dim: sides longer than it have no basis (QL or QR = I, no statistic; the published
 *   optimizer's maximum preconditioned dimension); 0 means 4096, the longest side a refresh takes.
 *   With both sides beyond it the step is AdamW.
 *   lr, weight_decay, shampoo_beta, shampoo_weight >= 0; beta1, beta2 in [0, 1); eps > 0;
 *   step t >= 1 (the bias-correction count); refresh 0/1; refresh_iters 1 .. 100;
 *   max_precond_dim 0 .. 4096. */
typedef struct {
  double lr;
  double weight_decay;
  double beta1;
  double beta2;
  double eps;
  double shampoo_beta;
  double shampoo_weight;
  int32_t step;
  int32_t refresh;
  int32_t refresh_iters;
  int32_t max_precond_dim;
} mfsdp_soap_hparams;

/* Bytes of device workspace mfsdp_soap_step needs for these entries and hyperparameters: per
 * matrix, zero-padded fp32 buffers of 8 mp np floats (mp, np = m, n rounded up to 128) and, per
 * side with a basis (padded length dp), 3 dp^2 + 640 dp + 17 * 128^2 floats: statistic, basis and
 * refresh product, and the QR's per-block reflectors and products (a side without a basis drops
 * all of these and, on the left, 2 mp np more); plus launch descriptors. Data pointers are not
 * used. 0 on invalid arguments; count == 0 returns 0 with no error. */
size_t mfsdp_soap_workspace_size(const mfsdp_soap_entry* entries, int64_t count,
                                 const mfsdp_soap_hparams* hp);

/* One SOAP step on every entry (host array of count entries), enqueued on `stream` (hipStream_t,
 * NULL = default stream); no host synchronisation. Every product runs at fp32 accuracy on the
 * bf16 MFMA as in mfsdp_shampoo_step (grouped over the entries); the refresh QR is a blocked
 * Householder factorization (16-column panels in 128-column blocks whose updates run on the same
 * GEMM). Part of each block update runs on a library-owned auxiliary stream of the current device
 * (default priority, created on first use, kept until the process ends), forked from `stream` and
 * joined back into it through events before the call returns, so `stream` orders everything the
 * call enqueues (and a graph captured from `stream` contains it). The workspace (device, 256-byte
 * aligned, >= the size query) must not be in use by another call still running. Returns MFSDP_OK,
 * MFSDP_E_INVALID, MFSDP_E_WORKSPACE or MFSDP_E_HIP; on an argument error nothing is enqueued.
 * At most 4096 entries per call. */
int mfsdp_soap_step(const mfsdp_soap_entry* entries, int64_t count, const mfsdp_soap_hparams* hp,
                    void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes for mfsdp_orthonormal_factor (0 on invalid arguments). */
size_t mfsdp_orthonormal_factor_workspace_size(int64_t d);

/* q = Q of the Householder QR decomposition a = Q R of a d x d fp32 matrix (row-major, device,
 * read only), with LAPACK's sign convention (the diagonal of R is -sign(pivot) times the column
 * norm; a column with nothing below its pivot gets the identity reflector): the factorization that
 * SOAP's basis refresh uses. 1 <= d <= 4096. `q` (d x d fp32, device) must not overlap `a`. Same
 * stream, workspace and error rules as mfsdp_soap_step. */
int mfsdp_orthonormal_factor(const float* a, float* q, int64_t d, void* workspace,
                             size_t workspace_bytes, void* stream);

/* ---- Owner planning (host only; no GPU, no stream) ---------------------------------------- */

/* Planner policies (Algorithm 1, "Balance-aware owner planning"). */
typedef enum {
  MFSDP_PLAN_ROLE_GREEDY = 0,   /* per block, in increasing block index, loads carried over */
  MFSDP_PLAN_SCOPE_GREEDY = 1,  /* the roles of all blocks pooled */
  MFSDP_PLAN_COST_AWARE = 2     /* scope plan if it balances strictly better within the cap */
} mfsdp_plan_policy;

/* One parameter of the sharded model, in the model's parameter order.
 *   block      index of its communication block (>= 0; blocks need not be contiguous)
 *   numel      element count (>= 0)
 *   is_matrix  1: a 2D matrix, one role of its own; 0: a non-2D tensor, packed with the block's
 *              other non-2D tensors into the block's one tail role (Section 4.1). */
typedef struct {
  int32_t block;
  int32_t is_matrix;
  int64_t numel;
} mfsdp_plan_param;

/* Owner rank of every parameter (Section 4.1, Algorithm 1): every role (a matrix, or a block's
 * tail) goes whole to one rank. Greedy rule: roles largest first, each to the currently lightest
 * rank (load = owned numel). ROLE_GREEDY runs it block by block in increasing block index, the
 * loads carried from block to block; SCOPE_GREEDY runs it once over all roles; COST_AWARE keeps the
 * SCOPE_GREEDY plan only if its largest rank load is strictly below ROLE_GREEDY's and, when
 * gamma_cap > 0, every block's gamma_B under it is <= gamma_cap; otherwise ROLE_GREEDY.
 * Ties (not fixed by the paper): roles of equal numel in the order (block, matrices before the
 * tail, first parameter index); among equally loaded ranks the lowest index.
 * gamma_B (Section 4.2 bandwidth model) = max_r O_{B,r} / (P_B / world), O_{B,r} the numel of
 * block B owned by rank r, P_B the block's numel; 0 for a block with P_B = 0.
 *   params, count     the parameters (host memory, read only); count == 0 is valid
 *   world             shard span W, 1 .. 65536
 *   policy            an mfsdp_plan_policy; gamma_cap is used by COST_AWARE only (<= 0: no cap)
 *   owner             out, count int32 owner ranks (host)
 *   rank_load         optional out (NULL = off), world int64 loads
 *   block_gamma       optional out, (1 + max block index) doubles
 *   policy_used       optional out, the policy whose plan was returned
 * Returns MFSDP_OK or MFSDP_E_INVALID (NULL, world out of range, unknown policy, NaN cap, negative
 * block or numel, is_matrix not 0/1); outputs are untouched on error. Thread safe; deterministic. */
int mfsdp_plan_owners(const mfsdp_plan_param* params, int64_t count, int32_t world, int32_t policy,
                      double gamma_cap, int32_t* owner, int64_t* rank_load, double* block_gamma,
                      int32_t* policy_used);

/* Per-block MatrixShard layouts of an owner plan (Section 4.1: a rank-indexed placement of each
 * flattened parameter interval; the last step of Algorithm 1: one layout per block, each validated
 * for one contiguous local segment per parameter). Layout rules (the paper fixes no packing order):
 * a block's canonical axis concatenates its parameters' elements in parameter order; rank r's
 * local buffer for block b holds the roles of b that r owns, ordered by each role's first parameter
 * index, a matrix whole and the block's tail as its non-2D tensors packed in parameter order; every
 * other rank's segment of a parameter is empty.
 *   params, count   as for mfsdp_plan_owners (host memory, read only); count == 0 is valid
 *   world           shard span, 1 .. 65536
 *   owner           count owner ranks (host, read only), e.g. from mfsdp_plan_owners
 *   global_offset   out, count int64: parameter i's offset on its block's canonical axis
 *   local_offset    out, count int64: parameter i's offset in its owner's local buffer of its block
 *   block_rank_len  optional out (NULL = off), (1 + max block index) * world int64: entry
 *                   b * world + r is rank r's local buffer length in block b
 * The emitted layout is validated (every rank's segments tile its local buffer of every block with
 * no gap or overlap, the tail is one packed segment, a block's local buffers add up to its
 * canonical axis). Returns MFSDP_OK or MFSDP_E_INVALID (NULL, world out of range, bad parameter,
 * owner out of range, a block's non-2D tensors with different owners, a failed validation); the
 * outputs are unspecified on error. Thread safe; deterministic; host only. */
int mfsdp_plan_layouts(const mfsdp_plan_param* params, int64_t count, int32_t world,
                       const int32_t* owner, int64_t* global_offset, int64_t* local_offset,
                       int64_t* block_rank_len);

/* Text for the last failure on the calling thread ("" if none). */
const char* mfsdp_last_error(void);
/* Name of a status code. */
const char* mfsdp_status_string(int status);
/* MFSDP_ABI_VERSION of the built library. */
int mfsdp_abi_version(void);
/* Identifier of the sources the library was built from (16 hex digits of a SHA-256 over its source
 * files, this header and the compiler flags, fixed at build time; "unknown" if the build did not set
 * it). Bindings compare it with the sources they ship to refuse a stale binary. Static string. */
const char* mfsdp_build_id(void);

#ifdef __cplusplus
}
#endif

#endif /* MFSDP_H */
