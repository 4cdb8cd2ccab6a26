/*
 * allegro_layer.h -- C ABI of one Allegro layer around the tensor product (gfx950).
 *
 * arxiv 2504.16068 names the parts of an Allegro layer without writing them
 * out: tensor features are mixed by the Clebsch-Gordan tensor product of
 * §II.D, scalar features are updated by MLPs, and every step runs in fp32
 * (Appendix, "Mixed-Precision Architecture"); Table I gives the model shapes
 * (rotation order, tensor features, number of layers).  The composition below
 * is this library's reading of that architecture, with the tensor product of
 * allegro_tp.h at its center.  Per edge e with center c(e):
 *
 *   1. environment weights     w[e,u]      = sum_l h[e,l] A[l,u]
 *   2. environment embedding   env         = allegro_env_embed(w, Y)
 *   3. tensor product          T           = allegro_tp_forward(V, env, W)
 *   4. per-irrep mixing        V'[e,v,k]   = sum_u Mix[c(k),v,u] T[e,u,k]
 *                              (c(k) = the x irrep that component k belongs to)
 *   5. invariant scalars       s[e,u]      = T[e,u,0]        (the 0e component)
 *   6. latent update           a           = [h, s] B1,   z = SiLU(a) = a / (1 + exp(-a)),
 *                              h'          = h + z B2
 *
 * Shapes: h, h' [E][L]; V, V', T [E][U][d1]; Y [E][d2]; A [L][U]; W [P][U];
 * Mix [n_x][U][U] (n_x = number of x irreps: 2(lmax+1) with full parity,
 * lmax+1 without); B1 [L+U][H]; B2 [H][L].  Sizes of the plan (lmax, parity,
 * U, d1, d2, P) come from allegro_tp.h.
 *
 * Supported: U = 64 (the tensor-feature count of the small and medium models
 * of Table I); L and H each 64 or 128; any lmax and parity of the plan.
 * Other shapes return ALLEGRO_E_UNSUPPORTED.
 *
 * Memory, ownership, execution and errors follow allegro_tp.h: caller-owned
 * row-major fp32 device memory, 16-byte aligned, no aliasing between inputs
 * and outputs, asynchronous on `stream`, no allocation per call, negative
 * codes with allegro_last_error().  The dense contractions (steps 1, 4 and 6
 * and their gradients) run on the fp32 matrix cores; the tensor product and
 * the embedding run the kernels of allegro_tp.h.  Every reduction over edges
 * has a fixed order, so results are bit-identical run to run.
 */
#ifndef ALLEGRO_LAYER_H
#define ALLEGRO_LAYER_H

#include <stddef.h>
#include <stdint.h>

#include "allegro_tp.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Device bytes of the two caller-owned buffers of one layer with N centers
 * and E edges:
 *   saved_bytes     activations the forward writes and the backward reads
 *                   (w, env, T, s, a);
 *   workspace_bytes scratch of the backward (its intermediate gradients and
 *                   the partial sums of its reductions).
 * Host-only; either output pointer may be NULL. */
int allegro_layer_buffers(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E,
                          size_t *saved_bytes, size_t *workspace_bytes);

/* Forward of one layer (steps 1-6): h_out [E][L] and V_out [E][U][d1] from
 * h [E][L], V [E][U][d1], Y [E][d2] and the weights A, W, Mix, B1, B2.
 * `saved` (at least saved_bytes of allegro_layer_buffers) receives the
 * activations that allegro_layer_backward needs; it is overwritten, and it
 * must stay untouched between the forward and its backward. */
int allegro_layer_forward(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E,
                          const int64_t *row_ptr, const float *h, const float *V, const float *Y,
                          const float *A, const float *W, const float *Mix, const float *B1,
                          const float *B2, float *h_out, float *V_out, void *saved,
                          size_t saved_bytes, void *stream);

/* VJP of one layer: given dh_out [E][L] and dV_out [E][U][d1] (the gradients
 * of a loss with respect to h_out and V_out), the gradients with respect to
 * the layer's inputs, dh [E][L], dV [E][U][d1], dY [E][d2], and to its
 * weights, dA [L][U], dW [P][U], dMix [n_x][U][U], dB1 [L+U][H], dB2 [H][L].
 * Inputs and weights are those of the forward, `saved` holds what that
 * forward wrote, and `workspace` (at least workspace_bytes of
 * allegro_layer_buffers) is overwritten.  Calls that share a saved buffer or
 * a workspace must not overlap.  With E == 0 every weight gradient is zero. */
int allegro_layer_backward(const allegro_tp_plan *plan, int L, int H, int64_t N, int64_t E,
                           const int64_t *row_ptr, const float *h, const float *V, const float *Y,
                           const float *A, const float *W, const float *Mix, const float *B1,
                           const float *B2, const void *saved, size_t saved_bytes,
                           const float *dh_out, const float *dV_out, float *dh, float *dV, float *dY,
                           float *dA, float *dW, float *dMix, float *dB1, float *dB2, void *workspace,
                           size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* ALLEGRO_LAYER_H */
