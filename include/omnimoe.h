/*
 * omnimoe.h - C ABI of the MI355X (gfx950) atomic-expert layer library (libomnimoe.so).
 *
 * The library computes the routed branch of the OmniMoE layer forward pass
 * (arXiv 2602.05711, "OmniMoE: An Efficient MoE by Orchestrating Atomic Experts at Scale"):
 *
 *   router    Cartesian Product Router, Sec. 2.2: row/column logits s_r = x W_r,
 *             s_c = x W_c per head (Eq. 9); the implicit grid S_ij = s_r[i] + s_c[j]
 *             (Eq. 11, with the LogSoftmax of Eq. 10 dropped: it shifts each half by a
 *             constant and changes neither the selection nor the gates); the top-K cells
 *             (Eq. 1) and softmax gates over their scores (Eq. 2).
 *   schedule  Expert-Centric Scheduling, Sec. 2.3: the T*H*K (token, expert) tasks
 *             (Eq. 12) sorted by (expert, task id), i.e. by (group, token) of Eq. 13 with
 *             groups of one active expert.
 *   experts   atomic experts E_e(x) = act(x . u_e) v_e (Eq. 4) with u = W[e], v = V[e]
 *             (Eq. 5-6), combined as y_t = sum over the token's (head, k) slots of
 *             g * act(x_t . u_e) * v_e (Eq. 7 without its shared MLP term; Eq. 14 per
 *             expert).
 *
 * Conventions
 *   - Tensor arguments are DEVICE pointers owned by the caller, row-major, contiguous.
 *     The library allocates no device memory: callers pass a workspace of at least
 *     omnimoe_workspace_size() bytes. The workspace and all outputs must not overlap
 *     the inputs or each other.
 *   - Every call is asynchronous on `stream` (a hipStream_t passed as void*; NULL is the
 *     default stream). The return value covers argument checks and launch errors; a
 *     fault inside a kernel surfaces at the caller's next synchronisation.
 *   - Pointers must be 16-byte aligned. Inputs must be finite.
 *   - Calls on different streams with different workspaces may run concurrently.
 *   - Indices: pair (task) p = (t * H + h) * K + k; expert id of grid cell (i, j) is
 *     n = i * n_cols + j; idx/gates are [T, H, K] with each (t, h) list ordered by
 *     score descending, ties to the lower expert id.
 */
#ifndef OMNIMOE_H
#define OMNIMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OMNIMOE_OK = 0,
  OMNIMOE_ERR_INVALID_ARG = 1, /* a size is out of range or a required pointer is NULL */
  OMNIMOE_ERR_UNSUPPORTED = 2, /* valid layer, but outside what the library implements */
  OMNIMOE_ERR_ALIGNMENT = 3,   /* a pointer is not 16-byte aligned */
  OMNIMOE_ERR_WORKSPACE = 4,   /* workspace smaller than omnimoe_workspace_size() */
  OMNIMOE_ERR_HIP = 5          /* the HIP runtime reported an error at launch */
} omnimoe_status;

typedef enum { OMNIMOE_F32 = 0, OMNIMOE_BF16 = 1 } omnimoe_dtype;
typedef enum { OMNIMOE_ACT_GELU = 0, OMNIMOE_ACT_SILU = 1 } omnimoe_act;
typedef enum { OMNIMOE_QUERY_SPLIT = 0, OMNIMOE_QUERY_SHARED = 1 } omnimoe_query_mode;

/* Layer shape. All sizes in elements.
 *   T           tokens; x is [T, d]. T = 0 is a valid no-op.
 *   d           hidden size; 8 <= d <= 8192, d % 8 == 0 (fp32 storage: d <= 4096, larger
 *               returns OMNIMOE_ERR_UNSUPPORTED).
 *   n_rows      N_r, rows of the expert grid; 1 <= n_rows <= 4096.
 *   n_cols      N_c, columns; 1 <= n_cols <= 4096. N = n_rows * n_cols experts.
 *   d_key       sub-key dimension; d_key % 8 == 0. SPLIT: rows score x[:, 0:d_key] and
 *               columns x[:, d_key:2 d_key] (2 d_key <= d). SHARED: both score
 *               x[:, 0:d_key] (d_key <= d).
 *   H           heads, each with its own sub-key tables, top-K and softmax; H >= 1.
 *   K           experts per (token, head); 1 <= K <= 4096 and K <= N (K > 64 selects
 *               with one workgroup per (token, head) instead of one wavefront; the dense
 *               router of the ablation takes K <= 64).
 *   dtype       storage type of x, sub-keys, u and v (OMNIMOE_F32 or OMNIMOE_BF16);
 *               arithmetic is fp32 in every case.
 *   act         activation of Eq. 4: GELU (erf form) or SiLU.
 *   query_mode  OMNIMOE_QUERY_SPLIT or OMNIMOE_QUERY_SHARED.
 *   group_size  B of Sec. 2.3, B >= 1: active experts per execution group. The schedule
 *               orders tasks by (group, task id) (Eq. 13); B = 1 gives (expert, task id).
 *               With B > 1 the layer computes the expert activations group by group as
 *               dense tiles on the matrix cores (Eq. 14, omnimoe_expert_forward_grouped)
 *               when dtype is bf16 and d % 64 == 0; its output then matches B = 1 to fp32
 *               rounding. Otherwise the output does not depend on B.
 * T * H * K and T * H * (n_rows + n_cols) must each be below 2^31. */
typedef struct {
  int64_t T;
  int32_t d;
  int32_t n_rows;
  int32_t n_cols;
  int32_t d_key;
  int32_t H;
  int32_t K;
  int32_t dtype;
  int32_t act;
  int32_t query_mode;
  int32_t group_size;
} omnimoe_layer_desc;

/* Stages, for workspace sizing and timing. */
typedef enum {
  OMNIMOE_STAGE_ROUTE = 0,
  OMNIMOE_STAGE_SELECT = 1,
  OMNIMOE_STAGE_SCHEDULE = 2,
  OMNIMOE_STAGE_EXPERT = 3,
  OMNIMOE_STAGE_LAYER = 4,
  OMNIMOE_STAGE_ROUTE_DENSE = 5,    /* omnimoe_route_dense without a logits buffer */
  OMNIMOE_STAGE_EXPERT_BACKWARD = 6, /* omnimoe_expert_backward */
  OMNIMOE_STAGE_ROUTE_BACKWARD = 7,  /* omnimoe_route_backward */
  OMNIMOE_STAGE_EXPERT_GROUPED = 8,  /* omnimoe_expert_forward_grouped */
  OMNIMOE_STAGE_EXPERT_SCATTER = 9,  /* omnimoe_expert_forward_scatter */
  OMNIMOE_STAGE_EXPERT_GROUP_ROWS = 10 /* omnimoe_expert_forward_group_rows */
} omnimoe_stage;

/* Bytes of workspace the given stage's entry point needs for this shape. */
omnimoe_status omnimoe_workspace_size(const omnimoe_layer_desc* desc, int32_t stage,
                                      size_t* bytes);

/* Router (Sec. 2.2; Eq. 9, 11, 1, 2).
 *   x            [T, d]                  dtype
 *   keys_row     [H, n_rows, d_key]      dtype   sub-keys of the grid rows (W_r^T per head)
 *   keys_col     [H, n_cols, d_key]      dtype   sub-keys of the grid columns
 *   idx          [T, H, K]  int32  out   selected expert ids, best first
 *   gates        [T, H, K]  fp32   out   softmax of the selected scores
 *   half_scores  [T, H, n_rows + n_cols] fp32 out, may be NULL: the row logits then the
 *                column logits of every (token, head), as computed on the way.
 * Logits accumulate in fp32 (MFMA for bf16). Selection compares those fp32 logits
 * exactly; a cell's score is their sum in double, which is exact. */
omnimoe_status omnimoe_route(const omnimoe_layer_desc* desc, const void* x, const void* keys_row,
                             const void* keys_col, int32_t* idx, float* gates, float* half_scores,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Dense router, the router ablation (Sec. 3.3, Table 3, "w/o Cartesian Product Router"):
 * every expert has its own gating vector and all N = n_rows * n_cols logits are computed.
 *   x        [T, d]      dtype
 *   w_gate   [H, N, d]   dtype   gating vector of every expert, per head
 *   idx      [T, H, K]   int32 out  top K by (logit descending, id ascending) (Eq. 1)
 *   gates    [T, H, K]   fp32  out  softmax of the K selected logits (Eq. 2)
 *   logits   [T, H, N]   fp32  out, may be NULL (then the workspace holds them:
 *            OMNIMOE_STAGE_ROUTE_DENSE bytes, T * H * N * 4 rounded up).
 * d_key and query_mode are not used. The logit GEMM accumulates in fp32 (MFMA for bf16). */
omnimoe_status omnimoe_route_dense(const omnimoe_layer_desc* desc, const void* x,
                                   const void* w_gate, int32_t* idx, float* gates, float* logits,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* The dense router's selection alone, from given fp32 logits [T, H, N]. */
omnimoe_status omnimoe_select_dense(const omnimoe_layer_desc* desc, const float* logits,
                                    int32_t* idx, float* gates, void* stream);

/* Selection only (Sec. 2.2, "Parallel Top-K Selection"; Eq. 11, 1, 2): for every (token, head)
 * row, the K best cells of the implicit grid S[i, j] = s_r[i] + s_c[j] (Eq. 11) by (S
 * descending, id ascending), id = i * n_cols + j (Eq. 1), and the softmax of their scores
 * (Eq. 2), from given fp32 logits
 *   half_scores [T, H, n_rows + n_cols] fp32   row logits then column logits (omnimoe_route's)
 *   idx         [T, H, K] int32 out,  gates [T, H, K] fp32 out   (as omnimoe_route's)
 * Comparisons are exact (S is the double sum of two floats), so the result depends only on
 * the logits. Needs no workspace (workspace may be NULL). */
omnimoe_status omnimoe_select(const omnimoe_layer_desc* desc, const float* half_scores,
                              int32_t* idx, float* gates, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Expert-Centric Scheduling (Sec. 2.3; Eq. 12-13).
 *   idx             [T, H, K] int32   expert ids in [0, N) (as from omnimoe_route)
 *   perm            [M] int32 out     task ids sorted by (expert, task id), M = T*H*K
 *   active          [min(M, N)] int32 out   distinct expert ids, ascending (first n_active used)
 *   active_offsets  [min(M, N) + 1] int32 out  active_offsets[a] = first position in perm of
 *                   expert active[a]; active_offsets[n_active] = M
 *   n_active        [1] int32 out (device)
 *   dense_offsets   [N + 1] int32 out, may be NULL: first position of every expert id
 *                   (the exclusive prefix sum of the per-expert task counts)
 * The result is unique, so it is the same on every run. */
omnimoe_status omnimoe_schedule(const omnimoe_layer_desc* desc, const int32_t* idx,
                                int32_t* perm, int32_t* active, int32_t* active_offsets,
                                int32_t* n_active, int32_t* dense_offsets, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Expert compute (Eq. 4, 7, 14) on a schedule.
 *   x      [T, d] dtype;  u, v  [N, d] dtype (down / up vectors of every expert)
 *   idx    [T, H, K] int32;  gates  [T, H, K] fp32;  perm  [M] int32 (from omnimoe_schedule)
 *   y      [T, d] fp32 out
 * Walks perm expert by expert: each expert's u row is read once per run of its tasks and
 * a[p] = g_p * act(x_t . u_e) is formed for each of them; then every token sums
 * a[p] * v_e over its slots in (head, k) order. When the routed pairs are dense (bf16, H = 1,
 * d % 64 == 0, K * 64 >= N, T * N * 2 bytes <= 16 GiB) the sum is instead one dense product
 * y = A V over all experts (Eq. 14 with a single group; A[t, e] = a[p] rounded to bf16), which
 * the workspace size accounts for. No atomics: y is the same on every run. */
omnimoe_status omnimoe_expert_forward(const omnimoe_layer_desc* desc, const void* x,
                                      const void* u, const void* v, const int32_t* idx,
                                      const float* gates, const int32_t* perm, float* y,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* Expert compute by groups of B active experts (Sec. 2.3, Eq. 13-14), desc->group_size = B:
 * for each group q, the activations G_q (.) act(X_q W_q^T) are computed as dense tiles on the
 * matrix cores, X_q being the distinct tokens of the group's tasks and W_q the u rows of its
 * experts, and only the entries that are tasks are kept, a[p] = g_p act(x_t . u_e); then
 * every token sums a[p] v_e over its slots in (head, k) order, as in omnimoe_expert_forward.
 * No atomics: y is the same on every run. It pays where the experts of a group share
 * tokens (many tasks per expert), and B = 1 is allowed but wastes the matrix cores.
 *   perm [M], active [min(M, N)], n_active [1] (device): omnimoe_schedule's outputs for the
 *   same desc (so the same group_size); group q holds the experts active[q B .. q B + B - 1],
 *   and perm lists its tasks in task order.
 * bf16 with d % 64 == 0, else OMNIMOE_ERR_UNSUPPORTED. omnimoe_layer_forward takes this path
 * whenever group_size > 1 and these hold. Results agree with omnimoe_expert_forward to fp32
 * rounding (the dot products are summed in another order). Workspace:
 * OMNIMOE_STAGE_EXPERT_GROUPED bytes. Pointers 16-byte aligned; T = 0 is a no-op. */
omnimoe_status omnimoe_expert_forward_grouped(const omnimoe_layer_desc* desc, const void* x,
                                              const void* u, const void* v, const int32_t* idx,
                                              const float* gates, const int32_t* perm,
                                              const int32_t* active, const int32_t* n_active,
                                              float* y, void* workspace, size_t workspace_bytes,
                                              void* stream);

/* Eq. 14 with both products group by group: the activations as in
 * omnimoe_expert_forward_grouped, then the second product (.)V_q per group. For every slot s
 * (a token t with tasks in group q, all of them adjacent in perm) a partial row
 * O[s] = sum over those tasks, in perm order, of a_p v_e (fp32, d wide), and then
 * y_t = sum of t's slot rows in group order. Arguments and layouts as
 * omnimoe_expert_forward_grouped (perm in (group, task id) order for desc->group_size).
 * The partial rows are written to and read back from the workspace: they move fewer bytes
 * than gathering v per task only when a token has many tasks per group (large groups, many
 * tasks per expert). bf16 and d % 64 == 0, else OMNIMOE_ERR_UNSUPPORTED. The result is the
 * same on every run. Workspace: OMNIMOE_STAGE_EXPERT_GROUP_ROWS bytes (the partial rows are
 * sized for min(M, ceil(min(M, N) / B) T) slots). */
omnimoe_status omnimoe_expert_forward_group_rows(const omnimoe_layer_desc* desc, const void* x,
                                                 const void* u, const void* v,
                                                 const int32_t* idx, const float* gates,
                                                 const int32_t* perm, const int32_t* active,
                                                 const int32_t* n_active, float* y,
                                                 void* workspace, size_t workspace_bytes,
                                                 void* stream);

/* Expert compute with the output stage in expert-major order, as the scatter-add of Eq. 14
 * orders it, made deterministic by a token-major reduction (the accumulate variant that reads
 * each v row once): a[p] = g_p * act(x_t . u_e) as in omnimoe_expert_forward; then, walking
 * perm expert by expert, each expert's v row is read once per run of its tasks and the fp32
 * row a[p] * v_e is written to row p of a contribution buffer [M, d] in the workspace; then
 * every token sums its H*K rows in (head, k) order into y. Same arguments as
 * omnimoe_expert_forward; workspace OMNIMOE_STAGE_EXPERT_SCATTER bytes (M * d * 4 for the
 * contribution rows plus M * 4). y agrees with omnimoe_expert_forward to fp32 rounding (each
 * product is rounded before it is added instead of fused into the sum) and is the same on
 * every run: no atomics. It exists to measure that trade-off: v is read A times instead of M
 * times, at the cost of writing and reading back M * d * 4 bytes. Pointers 16-byte aligned;
 * T = 0 is a no-op. */
omnimoe_status omnimoe_expert_forward_scatter(const omnimoe_layer_desc* desc, const void* x,
                                              const void* u, const void* v, const int32_t* idx,
                                              const float* gates, const int32_t* perm, float* y,
                                              void* workspace, size_t workspace_bytes,
                                              void* stream);

/* Expert compute without the schedule, token by token: the ablation of Expert-Centric
 * Scheduling (Sec. 3.3, Table 3, "w/o Expert-Centric Scheduling"), for measuring what the
 * schedule buys. Same arguments and result as omnimoe_expert_forward (bit for bit from 1024
 * tokens up; below that omnimoe_expert_forward adds each token's slots in four partial sums,
 * which can change the last bits), but every task gathers its own u and v rows: u is read once
 * per task, not once per expert run. Needs no workspace. Pointers 16-byte aligned; T = 0 is a
 * no-op. */
omnimoe_status omnimoe_expert_forward_token_centric(const omnimoe_layer_desc* desc,
                                                   const void* x, const void* u, const void* v,
                                                   const int32_t* idx, const float* gates,
                                                   float* y, void* stream);

/* Backward of the expert compute (gradients of Eq. 4 and 7) for a loss L with dL/dy = dy:
 *   h_p = x_t . u_e, a_p = g_p act(h_p), da_p = dy_t . v_e, dh_p = da_p g_p act'(h_p);
 *   dx       [T, d]  fp32 out   sum over t's slots of dh_p u_e (the expert branch's share of
 *                               dL/dx; the router's share is not included)
 *   du_rows  [n_active, d] fp32 out   row a: sum over the tasks of expert active[a] of
 *                               dh_p x_t (the gradient of u's row active[a]); min(M, N) rows
 *                               always suffice
 *   dv_rows  [n_active, d] fp32 out   row a: sum over those tasks of a_p dy_t
 *   dgates   [T, H, K] fp32 out   da_p act(h_p)
 *   dscores  [T, H, K] fp32 out   g_p (dgates_p - sum over the (t, h) row of g dgates): the
 *                               gradient of the K selected scores through the softmax (Eq. 2)
 * x, u, v, idx, gates as in omnimoe_expert_forward; dy [T, d] fp32; perm, active_offsets and
 * n_active from omnimoe_schedule with group_size 1 (each expert's tasks contiguous). The
 * per-expert sums run over the schedule's segments in task order, so the result is the same
 * on every run. d <= 4096 (bf16) or 2048 (fp32), else OMNIMOE_ERR_UNSUPPORTED. Workspace:
 * OMNIMOE_STAGE_EXPERT_BACKWARD bytes. */
omnimoe_status omnimoe_expert_backward(const omnimoe_layer_desc* desc, const void* x,
                                       const void* u, const void* v, const int32_t* idx,
                                       const float* gates, const int32_t* perm,
                                       const int32_t* active_offsets, const int32_t* n_active,
                                       const float* dy, float* dx, float* du_rows,
                                       float* dv_rows, float* dgates, float* dscores,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* Backward of the router's scores for fixed selections (the top-K choice is piecewise
 * constant, so gradients flow only through the selected scores S_p = s_r[i_p] + s_c[j_p],
 * Eq. 9 and 11), given dscores (as from omnimoe_expert_backward):
 *   dkeys_row [H, n_rows, d_key] fp32 out   row (h, i): sum over the tasks of head h whose
 *                                          expert lies in grid row i of dscores_p x_t[0:d_key]
 *   dkeys_col [H, n_cols, d_key] fp32 out   the same for grid columns, with x_t[c0:c0+d_key]
 *   dx        [T, d] fp32 in/out           adds sum over t's tasks of dscores_p keys_row[h, i_p]
 *                                          (columns 0:d_key) and dscores_p keys_col[h, j_p]
 *                                          (columns c0:c0+d_key); c0 = d_key (split) or 0
 * Tasks are sorted by sub-key with the schedule's radix sort and each sub-key's gradient is
 * summed over its tasks in task order, so the result is the same on every run. d_key <= 4096
 * (bf16) or 2048 (fp32), else OMNIMOE_ERR_UNSUPPORTED. Workspace: OMNIMOE_STAGE_ROUTE_BACKWARD
 * bytes. */
omnimoe_status omnimoe_route_backward(const omnimoe_layer_desc* desc, const void* x,
                                      const void* keys_row, const void* keys_col,
                                      const int32_t* idx, const float* dscores, float* dx,
                                      float* dkeys_row, float* dkeys_col, void* workspace,
                                      size_t workspace_bytes, void* stream);

/* The whole routed layer (Sec. 2.1-2.3): the routed term of Eq. 7, y_t = sum over heads h and
 * slots k of g_{t,h,k} act(x_t . u_e) v_e with e = idx[t, h, k] (Eq. 4-6), the experts and
 * gates chosen by the Cartesian Product Router (Eq. 9, 11, 1, 2) and the expert compute
 * ordered by Expert-Centric Scheduling (Eq. 12-14); on one stream, no host synchronisation.
 *   x [T, d], keys_row [H, n_rows, d_key], keys_col [H, n_cols, d_key], u, v [N, d]   dtype
 *   y [T, d] fp32 out; idx_out and gates_out ([T, H, K], as omnimoe_route's) may be NULL.
 * The expert compute is omnimoe_expert_forward's, or omnimoe_expert_forward_grouped's when
 * group_size > 1, dtype is bf16 and d % 64 == 0. With group_size 1, where the expert-major
 * order saves no memory traffic (at most 8192 tasks T*H*K, as in a decode step; at most one task
 * per two experts; or a u table N*d of at most 128 MiB, which stays in the GPU's last-level
 * cache), no schedule is formed: the same a_p are computed in slot order, with identical
 * results (by the selection kernel itself when there are at least 256 (token, head) rows;
 * omnimoe_layer_path tells which kernels run). With one head, K >= N / 64 and group_size 1,
 * both products run dense over all experts (Eq. 14 with a single group): x . u for every
 * (token, expert) pair, gate and activation kept at the selected pairs (a_p rounded to bf16),
 * then y = A V; no schedule is formed. Workspace:
 * OMNIMOE_STAGE_LAYER bytes
 * (caller-owned device memory, contents need not be initialised; OMNIMOE_ERR_WORKSPACE when
 * short). */
omnimoe_status omnimoe_layer_forward(const omnimoe_layer_desc* desc, const void* x,
                                     const void* keys_row, const void* keys_col, const void* u,
                                     const void* v, float* y, int32_t* idx_out, float* gates_out,
                                     void* workspace, size_t workspace_bytes, void* stream);

/* Which kernels omnimoe_layer_forward runs for a descriptor (no device work, no pointers):
 * *path receives an OR of the flags below. OMNIMOE_ERR_INVALID_ARG for a bad descriptor or a
 * NULL path. The result depends only on the descriptor, so it can be taken once per shape. */
typedef enum {
  OMNIMOE_PATH_SCHEDULE = 1,   /* the expert-major schedule is formed (Eq. 12-13); without it the
                                  a_p are formed in slot order */
  OMNIMOE_PATH_GROUPED = 2,    /* a_p from the grouped GEMM of Eq. 14 (group_size > 1) */
  OMNIMOE_PATH_SELECT_DOT = 4, /* the selection kernel also forms the slot-order a_p (no separate
                                  dot launch; the OMNIMOE_KERNEL_SELECT time includes it) */
  OMNIMOE_PATH_DENSE_SUM = 8,  /* the routed sum as one dense product over all experts (one head,
                                  K >= N / 64) */
  OMNIMOE_PATH_DENSE_DOT = 16  /* with groups of one expert, the a_p as well: x . u for every
                                  (token, expert) pair on the MFMA kernel, gate and activation
                                  kept at the selected pairs only (Eq. 14 with a single group;
                                  no schedule; OMNIMOE_KERNEL_SCHEDULE times the selection-mask
                                  pass, OMNIMOE_KERNEL_EXPERT_DOT this product) */
} omnimoe_path_flag;
omnimoe_status omnimoe_layer_path(const omnimoe_layer_desc* desc, int32_t* path);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): omnimoe_layer_forward with its workspace taken from
 * a scratch array of OMNIMOE_NOALLOC_SCRATCH_BYTES that the library holds in static device
 * memory, one per GPU, until the process ends. The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); the caller still passes inputs and outputs, with the
 * same meaning, layout and checks as omnimoe_layer_forward. It uses the scratch of the calling
 * thread's current device, which must be the device of `stream`; the first call on a device
 * looks the array's address up. A shape whose OMNIMOE_STAGE_LAYER workspace exceeds
 * OMNIMOE_NOALLOC_SCRATCH_BYTES returns OMNIMOE_ERR_WORKSPACE before any launch (at the
 * 1024 x 1024-expert, d = 2048, H = 8, K = 16 shape that is about 900 tokens). All calls on
 * one GPU share its array: calls that overlap in time on one GPU (other streams, other
 * threads) race and must be serialised by the caller. No state carries over between calls
 * (nothing in the scratch needs to start at zero). */
#define OMNIMOE_NOALLOC_SCRATCH_BYTES (64 * 1024 * 1024)
omnimoe_status omnimoe_layer_forward_noalloc(const omnimoe_layer_desc* desc, const void* x,
                                             const void* keys_row, const void* keys_col,
                                             const void* u, const void* v, float* y,
                                             int32_t* idx_out, float* gates_out, void* stream);

/* The shared dense branch MLP(x) that the full layer adds to the routed output (Eq. 3, 7),
 * as a SwiGLU feed-forward block of width d_ff:
 *   y[t] += w_down (silu(w_gu[0:d_ff] x_t) * (w_gu[d_ff:2 d_ff] x_t))
 *   x       [T, d]          dtype
 *   w_gu    [2 d_ff, d]     dtype   gate rows, then up rows
 *   w_down  [d, d_ff]       dtype
 *   y       [T, d]          fp32 in/out (e.g. the output of omnimoe_layer_forward)
 * d_ff % 8 == 0 and d_ff <= 65536 (else OMNIMOE_ERR_INVALID_ARG). Both projections accumulate
 * in fp32 on the logit GEMM kernels; silu(g) * u is rounded to the layer's dtype before the
 * down projection. Workspace: omnimoe_shared_mlp_workspace_size bytes. */
omnimoe_status omnimoe_shared_mlp_workspace_size(const omnimoe_layer_desc* desc, int32_t d_ff,
                                                 size_t* bytes);
omnimoe_status omnimoe_shared_mlp(const omnimoe_layer_desc* desc, int32_t d_ff, const void* x,
                                  const void* w_gu, const void* w_down, float* y,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* Per-kernel timing of omnimoe_layer_forward with HIP events on the call's stream.
 * A timer holds host-side state and HIP events only (no device memory). Kernel groups: */
typedef enum {
  OMNIMOE_KERNEL_SCORE = 0,      /* logit GEMM */
  OMNIMOE_KERNEL_SELECT = 1,     /* per-half top-K, Cartesian merge, gates */
  OMNIMOE_KERNEL_SCHEDULE = 2,   /* sort and segment kernels */
  OMNIMOE_KERNEL_EXPERT_DOT = 3, /* expert-major a = g * act(x . u) */
  OMNIMOE_KERNEL_ACCUMULATE = 4, /* token-major y = sum a * v */
  OMNIMOE_KERNEL_COUNT = 5
} omnimoe_kernel;

typedef struct omnimoe_timer omnimoe_timer;

/* capacity: how many timed calls may be recorded before omnimoe_timer_read. */
omnimoe_status omnimoe_timer_create(int32_t capacity, omnimoe_timer** timer);
omnimoe_status omnimoe_timer_destroy(omnimoe_timer* timer);
/* Waits for the recorded events, writes the summed milliseconds per kernel group
 * (ms[OMNIMOE_KERNEL_COUNT]) and the number of calls, and clears the timer. */
omnimoe_status omnimoe_timer_read(omnimoe_timer* timer, float* ms, int32_t* n_calls);
/* omnimoe_layer_forward with an event recorded around each kernel group. Returns
 * OMNIMOE_ERR_INVALID_ARG when the timer is full. */
omnimoe_status omnimoe_layer_forward_timed(const omnimoe_layer_desc* desc, const void* x,
                                           const void* keys_row, const void* keys_col,
                                           const void* u, const void* v, float* y,
                                           int32_t* idx_out, float* gates_out, void* workspace,
                                           size_t workspace_bytes, void* stream,
                                           omnimoe_timer* timer);

/* A static, human-readable name of a status code. */
const char* omnimoe_status_string(int32_t status);

#ifdef __cplusplus
}
#endif
#endif /* OMNIMOE_H */
