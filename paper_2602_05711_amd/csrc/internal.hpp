// Internal declarations shared by the host API and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace omnimoe {

// Derived sizes of one layer call (validated by the host API before any launch).
struct Shape {
  int64_t T;
  int d;
  int nr, nc;    // grid rows / columns
  int dk;        // sub-key dimension
  int H, K;
  bool bf16;     // storage type of x, keys, u, v
  int act;       // 0 GELU-erf, 1 SiLU
  int col0;      // first x column scored by the column half (d_key or 0)
  int64_t N;     // nr * nc
  int64_t M;     // T * H * K
  int64_t rows;  // T * H
  int hk;        // H * K
  int B;         // execution-group size of the schedule (Sec. 2.3)
};

// Logit GEMM: half_scores[t, h, 0:nr] = x[t, 0:dk] . keys_row[h, i, :],
// half_scores[t, h, nr:nr+nc] = x[t, col0:col0+dk] . keys_col[h, j, :].
// With accumulate, the products are added to half_scores instead of stored.
hipError_t launch_score(const Shape& s, const void* x, const void* keys_row,
                        const void* keys_col, float* half_scores, hipStream_t st,
                        bool accumulate = false);

// a[t, f] = silu(h[t, f]) * h[t, d_ff + f] for h [T, 2 d_ff] fp32; a [T, d_ff] in the layer's
// dtype (bf16 by round-to-nearest-even).
hipError_t launch_swiglu(int64_t T, int d_ff, bool bf16, const float* h, void* a,
                         hipStream_t st);

// Split-K bf16 product (fp32 out): out[z][m, n] = sum over k in [z kchunk, (z + 1) kchunk) of
// A[m, k] B[n, k], A [M, lda] and B [N, ldb] row-major, kchunk a multiple of 64, z < splits;
// partial z at out + z M N.
hipError_t launch_gemm_splitk(int64_t M, int N, const void* A, int64_t lda, const void* B,
                              int64_t ldb, int kchunk, int splits, float* out, hipStream_t st);

// The second product of Eq. 14 as one dense GEMM (all experts in one group), taken when
// dense_accumulate(s): bf16, one head, d % 64 == 0, K <= 4096, K * kDenseRatio >= N and the
// bf16 matrix A [T, N] within kDenseMaxBytes.
constexpr int64_t kDenseRatio = 64;
constexpr double kDenseMaxBytes = 16.0 * (1ull << 30);
bool dense_accumulate(const Shape& s);
size_t dense_accumulate_ws_bytes(const Shape& s);  // 0 when not taken
hipError_t launch_dense_accumulate(const Shape& s, const void* v, const int32_t* idx,
                                   const float* abuf, float* y, void* ws, hipStream_t st);

// The layer's first product over all experts as well (Eq. 14 with a single group), taken when
// dense_dot(s): dense_accumulate(s) with groups of one expert. launch_select_mask builds each
// token's selection mask and gates in expert-id order; launch_dense_dot runs h = X U^T with the
// masked-activation epilogue, leaving A at the start of ws; launch_dense_routed_sum then forms
// y = A V. ws holds dense_dot_ws_bytes(s) bytes for all three.
bool dense_dot(const Shape& s);
size_t dense_dot_ws_bytes(const Shape& s);  // 0 when not taken
hipError_t launch_select_mask(const Shape& s, const int32_t* idx, const float* gates, void* ws,
                              hipStream_t st);
hipError_t launch_dense_dot(const Shape& s, const void* x, const void* u, void* ws,
                            hipStream_t st);
hipError_t launch_dense_routed_sum(const Shape& s, const void* v, float* y, void* ws,
                                   hipStream_t st);

// bf16 product with the masked-activation epilogue: for t < T and n < ncols_out (a multiple of
// 64), aout[t, n] = bf16(g * act(x_t . u_n)) where bit n of sel_mask[t] is set (g =
// sel_gates[t, sel_pre[t, n / 32] + selected bits of that word below n]) and 0 elsewhere;
// x [T, d] and u [N, d] row-major, d % 64 == 0, no bit set at n >= N.
hipError_t launch_gemm_act_mask(int64_t T, int N, int ncols_out, const void* x, int d,
                                const void* u, const uint32_t* sel_mask, const int32_t* sel_pre,
                                int64_t words, const float* sel_gates, int hk, int act,
                                uint16_t* aout, hipStream_t st);

// Per-half top-K, Cartesian merge and gates from fp32 half-scores.
hipError_t launch_select(const Shape& s, const float* half_scores, int32_t* idx, float* gates,
                         hipStream_t st);

// launch_select followed by the slot-order dot of launch_slot_dot, in one kernel (the same idx,
// gates and a): bf16, K <= 64, nr == nc in {256, 512, 1024}, d / 8 in {64, 128, 256, 512}.
bool select_dot_fusable(const Shape& s);
hipError_t launch_select_dot(const Shape& s, const float* half_scores, int32_t* idx,
                             float* gates, const void* x, const void* u, float* abuf,
                             hipStream_t st);

// Dense-router selection (the router ablation): top K of each row of logits [rows, n] by
// (logit desc, id asc) and softmax gates.
hipError_t launch_select_dense(int64_t rows, int64_t n, int K, const float* logits, int32_t* idx,
                               float* gates, hipStream_t st);

// Radix-sort schedule. Workspace needs schedule_ws_bytes(M, N) bytes. On return sorted_keys
// points into the workspace (expert id of each sorted position), or is NULL when the groups
// hold more than one expert (then the expert of position i is idx[perm[i]]); with groups,
// *group_keys (if asked for) points to each sorted position's packed key
// (place of the expert in its group) << group_key_bits(s) | group.
size_t schedule_ws_bytes(int64_t M, int64_t N);
int group_key_bits(const Shape& s);
hipError_t launch_schedule(const Shape& s, const int32_t* idx, int32_t* perm, int32_t* active,
                           int32_t* active_offsets, int32_t* n_active, int32_t* dense_offsets,
                           void* ws, const int32_t** sorted_keys, hipStream_t st,
                           const int32_t** group_keys = nullptr);
// For the layer with groups of B > 1 experts: perm in (group, task id) order, active and
// n_active as launch_schedule gives them, *group_keys the sorted packed keys; no per-expert
// offsets. Same workspace as launch_schedule. Needs group_schedule_fits(s) (N <= 262144).
bool group_schedule_fits(const Shape& s);
hipError_t launch_group_schedule(const Shape& s, const int32_t* idx, int32_t* perm,
                                 int32_t* active, int32_t* n_active, void* ws,
                                 const int32_t** group_keys, hipStream_t st);

// a[p] = g_p * act(x_t . u_e) over the expert-major order given by perm (sorted_keys may be
// NULL: the kernel then reads idx[perm[pos]]).
hipError_t launch_expert_dot(const Shape& s, const void* x, const void* u, const int32_t* idx,
                             const float* gates, const int32_t* perm,
                             const int32_t* sorted_keys, float* a, hipStream_t st);

// dst[0:n] = value (a kernel, so the call can sit inside a captured graph).
hipError_t launch_fill_i32(int32_t* dst, int64_t n, int32_t value, hipStream_t st);

// The expert compute token by token (the scheduling ablation): same y as expert_dot followed
// by accumulate, with each task gathering its own u and v rows.
// Expert compute with per-task contribution rows: the expert dot into a[], then an
// expert-major pass writing c[p] = a[p] * v_e ([M, d] fp32) and a token-major sum of each
// token's rows in slot order into y.
hipError_t launch_expert_contrib(const Shape& s, const void* x, const void* u, const void* v,
                                 const int32_t* idx, const float* gates, const int32_t* perm,
                                 float* a, float* c, float* y, hipStream_t st);

hipError_t launch_token_centric(const Shape& s, const void* x, const void* u, const void* v,
                                const int32_t* idx, const float* gates, float* y,
                                hipStream_t st);

// Backward of the expert compute: dx, per-active-expert du / dv rows (expert-major, from a
// group-size-1 schedule), dgates and dscores. Workspace: backward_ws_bytes(M).
size_t backward_ws_bytes(int64_t M);
hipError_t launch_expert_backward(const Shape& s, const void* x, const void* u, const void* v,
                                  const int32_t* idx, const float* gates, const int32_t* perm,
                                  const int32_t* offsets, const int32_t* n_active,
                                  const float* dy, float* dx, float* du, float* dv,
                                  float* dgates, float* dscores, void* ws, hipStream_t st);

// Router backward for fixed selections: dkeys_row / dkeys_col written in full, dx added to.
size_t route_backward_ws_bytes(const Shape& s);
hipError_t launch_route_backward(const Shape& s, const void* x, const void* keys_row,
                                 const void* keys_col, const int32_t* idx, const float* dscores,
                                 float* dx, float* dkeys_row, float* dkeys_col, void* ws,
                                 hipStream_t st);

// Plan of the grouped expert GEMM (Eq. 14) over a schedule whose groups hold B > 1 active
// experts (tasks in (group, task id) order). A slot is a (group, token) pair; slots are numbered
// group by group, tokens ascending. Work tiles are 256 slots x grouped_tile_experts(B) experts
// of one group.
constexpr int kGroupSlots = 256;
int grouped_tile_experts(int B);
struct GroupPlan {
  const int32_t* key;   // [M]     packed key of sorted position i: place << gbits | group
  int gbits;
  int32_t* slot_token;  // [M]     token of slot s
  int32_t* slot_off;    // [M + 1] first sorted position of slot s (slot_off[slots] = M)
  int32_t* grp_slot;    // [G + 1] first slot of group q
  int32_t* grp_tile;    // [G + 1] first work tile of group q
  int32_t* counters;    // [0] slots, [1] work tiles
  int64_t G;            // upper bound on the number of groups: ceil(min(M, N) / B)
};
// sorted_group_keys: the schedule's packed keys, or NULL to derive them from perm, idx and
// active (a caller's schedule).
size_t group_plan_ws_bytes(const Shape& s);
hipError_t launch_group_plan(const Shape& s, const int32_t* perm, const int32_t* n_active,
                             const int32_t* sorted_group_keys, const int32_t* idx,
                             const int32_t* active, void* ws, GroupPlan* plan, hipStream_t st);

// Slots of a group plan in token order (stable: each token's slots in group order). slots[i]
// is a slot id, tokens[i] its token (T past the real slots), tok_start[t] the first place of
// token t (-1 when it has none). n >= the number of slots (the bound min(M, G T)).
struct SlotOrder {
  int32_t* slots;
  const int32_t* tokens;
  int32_t* tok_start;
};
size_t slot_sort_ws_bytes(int64_t n, int64_t T);
hipError_t launch_slot_sort(const GroupPlan& plan, int64_t n, int64_t T, void* ws,
                            SlotOrder* out, hipStream_t st);

// The second product of Eq. 14 group by group: O[s] = sum over the tasks of slot s, in
// position order, of a_p v_e (fp32 rows of d, n_slots_max of them), then y_t = sum of the
// token's slot rows in group order.
hipError_t launch_group_rows(const Shape& s, const void* v, const int32_t* idx,
                             const int32_t* perm, const float* a, const GroupPlan& plan,
                             const SlotOrder& order, float* rows, int64_t n_slots_max, float* y,
                             hipStream_t st);

// a[p] = g_p * act(x_t . u_e) by groups: per work tile, the 256 x 64 block of
// X_q U_q^T over the tile's slots (token rows) and experts on MFMA, then each task of the
// tile's slots whose expert lies in the tile reads its entry. bf16, d % 64 == 0.
hipError_t launch_grouped_dot(const Shape& s, const void* x, const void* u, const float* gates,
                              const int32_t* perm, const int32_t* active,
                              const int32_t* n_active, const GroupPlan& plan, float* a,
                              hipStream_t st);

// Where the expert-major order saves no memory traffic (M <= 8192, M <= N / 2, or a u table of
// at most 128 MiB): a[p] in slot order without a schedule (bf16 or fp32), identical to
// launch_expert_dot's a.
bool slot_dot(const Shape& s);
hipError_t launch_slot_dot(const Shape& s, const void* x, const void* u, const int32_t* idx,
                           const float* gates, float* abuf, hipStream_t st);

// y[t] = sum over slots (h, k) in order of a[p] * v[idx[p]].
hipError_t launch_accumulate(const Shape& s, const void* v, const int32_t* idx, const float* a,
                             float* y, hipStream_t st);

}  // namespace omnimoe
