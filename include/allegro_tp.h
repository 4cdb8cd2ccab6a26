/*
 * allegro_tp.h -- C ABI of the MI355X (gfx950) Allegro tensor-product library.
 *
 * The library computes, on one GPU, the operation that arxiv 2504.16068 names
 * the most expensive part of the Allegro architecture and accelerates with a
 * fused custom kernel (§II.D "Optimized Tensor Product Kernel"): the per-edge,
 * channel-wise Clebsch-Gordan tensor product, its first derivative (the VJP
 * that inference-time forces need, §II.D), and the environment embedding the
 * product consumes.  The coupling coefficients are held in the compressed
 * sparse "combined tensor of Wigner 3-j coefficients" form the paper describes
 * (§II.D, last paragraph), and the outer product of the two inputs is never
 * materialised (same paragraph).  Arithmetic is fp32, as the paper's
 * mixed-precision scheme prescribes for tensor products (Appendix,
 * "Mixed-Precision Architecture").
 *
 * Notation
 *   N      atoms (centers), E edges, U channels ("tensor features", Table I)
 *   lmax   maximum rotation order (Table I: 2 or 3)
 *   x / out irreps: for l = 0..lmax, (l, (-1)^l) and, with full parity, also
 *          (l, -(-1)^l); components m = -l..l; blocks concatenated -> d1
 *   env irreps: (l, (-1)^l) for l = 0..lmax -> d2 = (lmax+1)^2
 *   paths: every (a, b, c) with |l_a - l_b| <= l_c <= l_a + l_b and
 *          p_c = p_a p_b, ordered lexicographically by (a, b, c) -> P
 *   CSR:   edges sorted by center; edge e belongs to center n iff
 *          row_ptr[n] <= e < row_ptr[n+1]; c(e) is that n.
 *
 * Operations (exact definitions; the kernels reach the same values up to fp32
 * rounding order):
 *   env[n,u,j]   = sum_{e in seg(n)} w[e,u] Y[e,j]
 *   out[e,u,k]   = sum_p W[p,u] sum_{(i,j,k) in p} C_ijk x[e,u,i] env[c(e),u,j]
 *   grad_x[e,u,i]   = sum_p W[p,u] sum C_ijk env[c(e),u,j] g[e,u,k]
 *   grad_env[n,u,j] = sum_{e in seg(n)} sum_p W[p,u] sum C_ijk x[e,u,i] g[e,u,k]
 *   grad_w[e,u]     = sum_j grad_env[c(e),u,j] Y[e,j]
 *   grad_Y[e,j]     = sum_u grad_env[c(e),u,j] w[e,u]
 *   C is the real coupling tensor of each path, orthonormal in (m1, m2) for
 *   every m3 and signed so that its first non-zero entry (row-major m1, m2,
 *   m3) is positive; real components follow the real spherical harmonics with
 *   l = 1 ordered (y, z, x).
 *
 * Memory and ownership
 *   Every tensor argument is a device pointer to caller-owned, row-major,
 *   contiguous fp32 (int64 for row_ptr) memory, 16-byte aligned.  Outputs are
 *   fully overwritten (never accumulated) and must not alias any input or each
 *   other.  The library never allocates or frees caller memory and allocates
 *   nothing per call; a plan owns at most a 4-byte device status word.
 *
 * Execution
 *   Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *   stream) and do not synchronise, except under ALLEGRO_VALIDATE.  A plan is
 *   immutable after creation, so calls with one plan on different streams may
 *   run concurrently.
 *
 * Errors
 *   Every entry point returns ALLEGRO_OK (0) or a negative code and then sets
 *   a thread-local message readable with allegro_last_error().  Host checks:
 *   null pointers, misalignment, N < 0, E < 0, E > 0 with N == 0, N >= 2^31,
 *   unsupported lmax / U.  E == 0 and N == 0 is a successful no-op; E == 0
 *   with N > 0 writes zero env / grad_env.  Launch failures give
 *   ALLEGRO_E_HIP.  With ALLEGRO_VALIDATE the call also checks on the device
 *   that row_ptr[0] == 0, row_ptr[N] == E and row_ptr is non-decreasing, and
 *   waits for that check (and only then launches the operation).
 */
#ifndef ALLEGRO_TP_H
#define ALLEGRO_TP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct allegro_tp_plan allegro_tp_plan;

enum {
  ALLEGRO_OK = 0,
  ALLEGRO_E_INVALID = -1,     /* bad argument (pointer, size, alignment, CSR) */
  ALLEGRO_E_UNSUPPORTED = -2, /* lmax or U outside the compiled set */
  ALLEGRO_E_HIP = -3,         /* HIP runtime or launch failure */
  ALLEGRO_E_NOMEM = -4,       /* plan allocation failed */
  ALLEGRO_E_TIMEOUT = -5      /* a bounded wait on the device ran out (reported under ALLEGRO_VALIDATE) */
};

enum {
  ALLEGRO_FULL_PARITY = 1,   /* x / out carry both parities per l (else natural parity only) */
  ALLEGRO_DETERMINISTIC = 2, /* env: fixed ascending-edge fp32 order, no fused multiply-add */
  ALLEGRO_VALIDATE = 4       /* device-side CSR check before each call (synchronises) */
};

/* Create a plan for maximum rotation order lmax (1, 2 or 3), U channels
 * (16, 32, 64 or 128) and flags (ALLEGRO_*).  Builds the sparse coupling table
 * on the host; only with ALLEGRO_VALIDATE does it touch the GPU, to allocate
 * the plan's 4-byte device status word.  *plan is set to NULL on failure; a
 * failed allocation returns ALLEGRO_E_NOMEM.  For tests of that path, the
 * environment variable ALLEGRO_SIMULATE_ALLOC_FAILURE set to "plan", "table"
 * or "status" makes that allocation fail (the status word's without calling
 * HIP). */
int allegro_tp_plan_create(allegro_tp_plan **plan, int lmax, int U, int flags);

/* Release a plan (NULL is accepted). The caller must ensure no call using it
 * is still running on any stream. */
int allegro_tp_plan_destroy(allegro_tp_plan *plan);

/* Sizes of a plan: d1 (x / out components), d2 (env components), number of
 * paths and number of non-zero coupling coefficients.  Any output pointer may
 * be NULL.  path_desc, if not NULL, receives n_paths rows of 6 ints
 * (l1, p1, l2, p2, l3, p3) in path order (p = +1 even, -1 odd). */
int allegro_tp_plan_query(const allegro_tp_plan *plan, int *d1, int *d2, int *n_paths,
                          int *path_desc, int *nnz);

/* Copy the plan's sparse combined coupling table to host memory:
 * idx receives nnz rows of (path, i, j, k) -- i / k index x / out components,
 * j env components -- and val the coefficients in fp64.  Both are caller-owned
 * host arrays of at least 4 * nnz ints and nnz doubles. */
int allegro_tp_plan_cg(const allegro_tp_plan *plan, int *idx, double *val);

/* Environment embedding: env[N][U][d2] from w[E][U] and Y[E][d2].
 * With ALLEGRO_DETERMINISTIC each env value is the strict left-to-right fp32
 * sum over the segment of the fp32-rounded products (no FMA), bit-identical
 * run to run; otherwise FMA contraction is used (still a fixed order). */
int allegro_env_embed(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                      const float *w, const float *Y, float *env, void *stream);

/* Tensor product forward: out[E][U][d1] from x[E][U][d1], env[N][U][d2] and
 * path weights path_w[P][U] (a scalar per path is passed broadcast over U). */
int allegro_tp_forward(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                       const float *x, const float *env, const float *path_w, float *out,
                       void *stream);

/* Tensor product VJP plus the embedding's VJP, given grad_out[E][U][d1]:
 * grad_x[E][U][d1], grad_env[N][U][d2], and through the embedding
 * grad_w[E][U] and grad_Y[E][d2] (w and Y are the embedding's inputs).
 * No path-weight gradient is computed. */
int allegro_tp_backward(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                        const float *x, const float *env, const float *path_w,
                        const float *grad_out, const float *w, const float *Y,
                        float *grad_x, float *grad_env, float *grad_w, float *grad_Y,
                        void *stream);

/* Bytes of device workspace that allegro_tp_backward_train needs for N centers:
 * (N + 128) * n_paths * U floats at lmax < 3; at lmax 3 max(1, min(N, 1024)) *
 * n_paths * U floats (a bound on the matrix-core kernel's per-wave rows that
 * holds on any device).  Host-only; no GPU needed. */
int allegro_tp_backward_workspace(const allegro_tp_plan *plan, int64_t N, size_t *bytes);

/* Training backward: everything allegro_tp_backward computes, plus the
 * gradient of the path weights (needed to train them; the paper leaves the
 * training kernels to future work, §II.D):
 *   grad_path_w[p][u] = sum_e sum_{(i,j,k) in p} C_ijk x[e,u,i] env[c(e),u,j] grad_out[e,u,k]
 * (for one scalar weight per path, sum grad_path_w over u).  The sum is
 * deterministic.  At lmax < 3 each center's contribution is summed over its
 * edges in a fixed order and written to one workspace row of n_paths * U
 * floats per center (path-major), which two reduction launches then sum in a
 * fixed order.  At lmax 3 each wave of the matrix-core kernel keeps one
 * channel group and sums the contributions of the centers it visits, in
 * order, into one channel-major workspace row of its own (R rounds of U rows
 * of n_paths floats, R = its wave count over U / channels per wave: 16 on a
 * 256-compute-unit MI355X at U = 128); one launch sums the R rounds in order.
 * The grid is fixed per device, so the result is bit-identical run to run on
 * one device.  The other four gradients
 * equal allegro_tp_backward's up to fp32 rounding (the two split the work
 * differently; at lmax 3 this call forms grad_x = M^T grad_out with the
 * per-center matrix of the forward).  workspace is caller-owned device memory of at least
 * allegro_tp_backward_workspace() bytes, 16-byte aligned, overwritten (no
 * clearing needed); calls that share a workspace must not overlap.  N == 0
 * sets grad_path_w to zero.  Errors as for allegro_tp_backward, plus
 * ALLEGRO_E_INVALID for a missing or too small workspace.  At lmax 3 the
 * matrix-core kernel's waves hand work to each other through bounded waits
 * (about a second each); one that ran out (a stalled wave; it does not happen
 * in a working kernel) makes the kernel finish without waiting further, and
 * its outputs are then not valid: with ALLEGRO_VALIDATE the call waits for the
 * kernel and returns ALLEGRO_E_TIMEOUT.  For tests of that path, a plan
 * created while the environment variable ALLEGRO_SIMULATE_HANDOVER_TIMEOUT is
 * set gives up every such wait at once. */
int allegro_tp_backward_train(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                              const float *x, const float *env, const float *path_w,
                              const float *grad_out, const float *w, const float *Y,
                              float *grad_x, float *grad_env, float *grad_w, float *grad_Y,
                              float *grad_path_w, void *workspace, size_t workspace_bytes,
                              void *stream);

/* Allocation-free training backward, for callers that cannot allocate device
 * memory or pass a workspace (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): the same outputs as
 * allegro_tp_backward_train, with the path-weight partial sums kept in a
 * static device array of the library instead of a workspace.  The array is
 * 64 MiB of fp32 (16 Mi floats) and is held by every GPU the library runs on
 * until the process ends.  At lmax 3 the matrix-core kernel's per-wave rows
 * (at most 1024 x U x n_paths floats) fit it at any N: one launch and the
 * same reduction as allegro_tp_backward_train, whose outputs it reproduces
 * bit for bit.  At lmax < 3 the centers are processed in chunks of
 * C = floor(16 Mi / (n_paths * U)) - 384 centers (8,354 at lmax 2, U = 64);
 * each chunk's per-center rows are summed in a fixed order into one row, and
 * the chunk rows in order into grad_path_w, so the result is deterministic and
 * equals allegro_tp_backward_train's up to fp32 rounding order (grad_x,
 * grad_env, grad_w and grad_Y are bit-identical to it); at most 256 chunks:
 * N > 256 * C returns ALLEGRO_E_INVALID before any launch.  Every call on one GPU shares that GPU's array and overwrites it, so
 * calls that overlap on one GPU (several streams or threads) race and must be
 * serialised by the caller.  The call itself allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); the first call on a device looks the
 * array's address up there (hipGetSymbolAddress).  Errors as for
 * allegro_tp_backward_train. */
int allegro_tp_backward_train_noalloc(const allegro_tp_plan *plan, int64_t N, int64_t E, const int64_t *row_ptr,
                                      const float *x, const float *env, const float *path_w,
                                      const float *grad_out, const float *w, const float *Y,
                                      float *grad_x, float *grad_env, float *grad_w, float *grad_Y,
                                      float *grad_path_w, void *stream);

/* Real spherical harmonics of the edge vectors, the embedding input of the
 * environment sum (Appendix "Mixed-Precision Architecture": embedded in fp64,
 * then cast to fp32): Y[E][d2] = fl32(Y^l_m(vec_e)), l = 0..lmax, m = -l..l,
 * component normalisation sum_m (Y^l_m)^2 = 2l + 1, real basis with l = 1
 * ordered (y, z, x).  vec[E][3] is fp64 (r_ij = r_j - r_i); Y depends on its
 * direction only.  A zero vector has no direction and yields NaN. */
int allegro_sh_forward(const allegro_tp_plan *plan, int64_t E, const double *vec, float *Y, void *stream);

/* VJP of allegro_sh_forward, in fp64 as the forward: grad_vec[e][k] =
 * sum_j grad_Y[e][j] dY_j/dvec_e[k], with grad_Y[E][d2] fp32 (as produced by
 * allegro_tp_backward) and grad_vec[E][3] fp64.  Summing grad_vec into the two
 * atoms of each edge (minus at the center, plus at the neighbour) gives that
 * loss's gradient with respect to positions through the harmonics. */
int allegro_sh_backward(const allegro_tp_plan *plan, int64_t E, const double *vec, const float *grad_Y,
                        double *grad_vec, void *stream);

/* Message of the last failed call on this thread ("" if none). */
const char *allegro_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ALLEGRO_TP_H */
