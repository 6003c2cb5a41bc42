/*
 * Oracle for the OmniMoE atomic-expert layer forward pass: TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, host-only implementation in double precision, written from the
 * paper (arXiv 2602.05711, "OmniMoE"). It exists to check the GPU library and is
 * used only by the tests, the smoke check and the CPU-baseline leg of the
 * benchmark. It shares no source with the GPU library.
 *
 * Inputs are float32 host arrays (bf16 inputs are passed as their exact float32
 * widening). Layouts:
 *   x          [T, d]
 *   keys_row   [H, n_rows, d_key]      sub-keys scoring grid rows
 *   keys_col   [H, n_cols, d_key]      sub-keys scoring grid columns
 *   u, v       [N, d], N = n_rows * n_cols   down (w_in) and up (w_out) vectors
 *   idx/gates  [T, H, K]               pair p = (t * H + h) * K + k
 * Expert id of grid cell (i, j) is n = i * n_cols + j.
 *
 * Every function returns 0 on success and a negative value on bad arguments.
 */
#ifndef OMNIMOE_REF_H
#define OMNIMOE_REF_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int64_t T;
  int32_t d;
  int32_t n_rows;
  int32_t n_cols;
  int32_t d_key;
  int32_t H;
  int32_t K;
  int32_t act;        /* 0: GELU (erf form), 1: SiLU */
  int32_t query_mode; /* 0: split (rows read x[0:d_key], columns x[d_key:2 d_key]); 1: shared (both x[0:d_key]) */
  int32_t group_size; /* B >= 1: active experts per execution group */
} omnimoe_ref_desc;

/* Row and column logits s_r = x W_r, s_c = x W_c per head (Eq. 9), fp64, summed
 * over the key dimension in ascending order. sr [T, H, n_rows], sc [T, H, n_cols]. */
int omnimoe_ref_half_scores(const omnimoe_ref_desc* desc, const float* x, const float* keys_row,
                            const float* keys_col, double* sr, double* sc, int n_threads);

/* Top-K over the implicit score grid S_ij = sr[i] + sc[j] (Eq. 11), order
 * (S descending, n ascending), and softmax gates over the K selected scores
 * (Eq. 2). method 0: brute force over all N cells (the definition, Eq. 1);
 * method 1: per-half top-K then the Cartesian candidates (a+1)(b+1) <= K;
 * method 2: brute force on the literal LogSoftmax log-probabilities of Eq. 10.
 * sel_scores receives the selected S values (may be NULL). Returns the number of
 * candidate sums that were not exact in double (see omnimoe_ref.cpp) in
 * *inexact_sums when that pointer is not NULL. */
int omnimoe_ref_select(const omnimoe_ref_desc* desc, const double* sr, const double* sc,
                       int method, int32_t* idx, double* sel_scores, double* gates,
                       int64_t* inexact_sums, int n_threads);

/* Same selection starting from float32 half-scores laid out [T, H, n_rows + n_cols]
 * (row logits first), as produced by the GPU scoring stage. */
int omnimoe_ref_select_f32(const omnimoe_ref_desc* desc, const float* half_scores, int method,
                           int32_t* idx, double* sel_scores, double* gates,
                           int64_t* inexact_sums, int n_threads);

/* Expert-Centric Scheduling (Eq. 12-13): pairs sorted by (group of the active
 * expert, pair id). perm [M]; active [<= min(M, N)] ascending expert ids;
 * active_offsets [n_active + 1] first sorted position of each active expert,
 * last entry M; dense_offsets [N + 1] (may be NULL) first sorted position of
 * expert e. M = T * H * K, N = n_rows * n_cols. */
int omnimoe_ref_schedule(const omnimoe_ref_desc* desc, const int32_t* idx, int32_t* perm,
                         int32_t* active, int32_t* active_offsets, int32_t* n_active,
                         int32_t* dense_offsets);

/* Routed output y[t] = sum over (h, k) of g * act(x_t . u_e) * v_e (Eq. 4, 7),
 * fp64. scheduled = 0 walks tokens in order; scheduled = 1 walks the expert-major
 * schedule to form a[p] = g_p * act(x_t . u_e) and then sums a[p] * v_e per
 * token in slot order. The two give bit-identical y. gates are fp64 [T, H, K]. */
int omnimoe_ref_expert_forward(const omnimoe_ref_desc* desc, const float* x, const float* u,
                               const float* v, const int32_t* idx, const double* gates,
                               int scheduled, double* y, int n_threads);

/* Whole layer: half-scores, selection (method as above), schedule, scheduled
 * forward. idx, gates may be NULL. */
int omnimoe_ref_layer_forward(const omnimoe_ref_desc* desc, const float* x, const float* keys_row,
                              const float* keys_col, const float* u, const float* v, int method,
                              double* y, int32_t* idx, double* gates, int n_threads);

/* Dense router, the router ablation (Sec. 3.3, Table 3, "w/o Cartesian Product Router"):
 * logits L[t, h, n] = x_t . w_gate[h, n] over all N = n_rows * n_cols experts (fp64,
 * summed over d in ascending order), top-K by (L descending, n ascending) (Eq. 1) and
 * softmax gates over the K selected logits (Eq. 2). w_gate [H, N, d]; idx, gates [T, H, K];
 * logits [T, H, N] may be NULL. d_key and query_mode are not used. */
int omnimoe_ref_route_dense(const omnimoe_ref_desc* desc, const float* x, const float* w_gate,
                            int32_t* idx, double* gates, double* logits, int n_threads);

/* The dense router's selection from given float32 logits [T, H, N]. */
int omnimoe_ref_select_dense_f32(const omnimoe_ref_desc* desc, const float* logits,
                                 int32_t* idx, double* gates, int n_threads);

/* The shared dense branch MLP(x) of Eq. 3 / Eq. 7, as a SwiGLU feed-forward block:
 *   g_f = x . w_gu[f],  u_f = x . w_gu[d_ff + f]  (f < d_ff),  a_f = silu(g_f) * u_f,
 *   y[t, c] += sum_f w_down[c, f] * a_f            (fp64, sums in ascending index order).
 * w_gu [2 d_ff, d] (gate rows, then up rows); w_down [d, d_ff]; y [T, d] is added to. */
int omnimoe_ref_shared_mlp(const omnimoe_ref_desc* desc, int32_t d_ff, const float* x,
                           const float* w_gu, const float* w_down, double* y, int n_threads);

/* Backward of the expert compute (the gradients of Eq. 4 / 7 for L = sum_t dy_t . y_t), fp64:
 *   h_p = x_t . u_e, a_p = g_p act(h_p), da_p = dy_t . v_e,
 *   dgates[p]  = da_p act(h_p)
 *   dscores[p] = g_p (dgates[p] - sum over the K slots q of (t, h) of g_q dgates[q])
 *                (the gradient with respect to the selected scores through the softmax, Eq. 2)
 *   dx[t]      = sum over t's slots of da_p g_p act'(h_p) u_e
 *   du_rows[a] = sum over the tasks of expert active[a] of da_p g_p act'(h_p) x_t
 *   dv_rows[a] = sum over the tasks of expert active[a] of a_p dy_t
 * Rows of du / dv are those of the active experts in ascending id order (active[a], a <
 * *n_active); x, u, v fp32 as stored, gates and dy fp64. */
int omnimoe_ref_expert_backward(const omnimoe_ref_desc* desc, const float* x, const float* u,
                                const float* v, const int32_t* idx, const double* gates,
                                const double* dy, double* dx, double* du_rows, double* dv_rows,
                                int32_t* active, int32_t* n_active, double* dgates,
                                double* dscores, int n_threads);

/* Backward of the router's scores for fixed selections (the selection itself is piecewise
 * constant): with S_p = s_r[t, h, i_p] + s_c[t, h, j_p] (Eq. 9, 11) and dL/dS_p = dscores[p],
 *   dkeys_row[h, i] = sum over tasks p of (t, h) with row i_p = i of dscores[p] x_t[0 : d_key]
 *   dkeys_col[h, j] = sum over tasks with column j_p = j of dscores[p] x_t[c0 : c0 + d_key]
 *   dx[t]          += sum over t's tasks of dscores[p] (keys_row[h, i_p] on x[0 : d_key] and
 *                     keys_col[h, j_p] on x[c0 : c0 + d_key])
 * (c0 = d_key for split queries, 0 for shared). dkeys_row [H, n_rows, d_key] and dkeys_col
 * [H, n_cols, d_key] are written in full; dx [T, d] is added to. fp64. */
int omnimoe_ref_route_backward(const omnimoe_ref_desc* desc, const float* x, const float* keys_row,
                               const float* keys_col, const int32_t* idx, const double* dscores,
                               double* dx, double* dkeys_row, double* dkeys_col, int n_threads);

/* Derivative of the activation on one value: 0 GELU-erf, 1 SiLU. */
double omnimoe_ref_act_grad(int act, double z);

/* The activation on one value: 0 GELU-erf, 1 SiLU. */
double omnimoe_ref_act(int act, double z);

#ifdef __cplusplus
}
#endif
#endif
