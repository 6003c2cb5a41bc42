// Backward of the expert compute (Eq. 4, 7) for L = sum_t dy_t . y_t, the gradients a training
// step needs from this layer's experts and gates:
//   h_p = x_t . u_e,  a_p = g_p act(h_p),  da_p = dy_t . v_e,
//   dgates_p = da_p act(h_p),  dh_p = da_p g_p act'(h_p),
//   dx_t = sum over t's slots of dh_p u_e,
//   du_e = sum over e's tasks of dh_p x_t,  dv_e = sum over e's tasks of a_p dy_t,
//   dscores_p = g_p (dgates_p - sum over the (t, h) row of g dgates)   (softmax, Eq. 2).
// token pass: one wavefront per token gathers each slot's u and v rows (as the token-centric
//   forward does), forms h, da, a, dh, dgates and sums dx in slot order;
// expert pass: one wavefront per active expert walks its segment of the schedule (task ids
//   ascending) and sums du and dv in that order: the expert-major order makes the per-expert
//   gradients plain sequential sums, with no atomics, so every run gives the same bits;
// score pass: one wavefront per (token, head) row.
// Router backward (selections fixed; S_p = s_r[i_p] + s_c[j_p]): tasks are sorted by sub-key
// row (h, i) with the schedule's radix sort, and one wavefront per selected sub-key sums
// dscores_p x_t over its segment in task order (the same expert-major pattern, applied to the
// sub-key tables); the input gradient adds dscores_p times the two sub-keys, token by token.
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

struct BwdArgs {
  const void* x;
  const void* u;
  const void* v;
  const int32_t* idx;
  const float* gates;
  const float* dy;
  const int32_t* perm;
  const int32_t* offsets;
  const int32_t* n_active;
  float* dx;
  float* du;
  float* dv;
  float* dgates;
  float* dscores;
  float* a;    // a_p per task (workspace)
  float* dh;   // dh_p per task (workspace)
  int64_t T;
  int64_t N;
  int64_t M;
  int64_t cap;  // min(M, N): rows of du / dv
  int d;
  int hk;
  int K;
  int act;
  int nchunks;  // 16-byte chunks of a stored row
};

__device__ __forceinline__ int clamp_id(int v, int64_t n) {
  return v < 0 ? 0 : (v >= n ? (int)(n - 1) : v);
}

// Element k (0 .. EPC-1) of a stored 16-byte chunk, as fp32.
template <bool BF16>
__device__ __forceinline__ float chunk_elem(const uint4& c, int k) {
  if constexpr (BF16) {
    const uint32_t w = k < 2 ? c.x : (k < 4 ? c.y : (k < 6 ? c.z : c.w));
    return (k & 1) ? bf16_hi(w) : bf16_lo(w);
  } else {
    const uint32_t w = k == 0 ? c.x : (k == 1 ? c.y : (k == 2 ? c.z : c.w));
    return __uint_as_float(w);
  }
}

// Slots s0 .. s0 + GG - 1 of token t (expert e and gate g of slot s0 + i on lane i of ev/gv, an
// offset of the slot batch sb): their u and v rows are loaded together, then h, da, a, dh and
// dgates are formed and dx += dh u_e summed in slot order.
template <int GG, int CPL, bool BF16>
__device__ __forceinline__ void token_slots(const BwdArgs& a, int64_t t, int s0, int sb, int ev,
                                            float gv, const uint4 (&xr)[CPL],
                                            const float (&dyr)[CPL][BF16 ? 8 : 4],
                                            const bool (&cv)[CPL],
                                            float (&acc)[CPL][BF16 ? 8 : 4]) {
  constexpr int EPC = BF16 ? 8 : 4;
  const int l = lane_id();
  const uint4* U = (const uint4*)a.u;
  const uint4* V = (const uint4*)a.v;
  const int64_t rc = a.nchunks;
  uint4 ur[GG][CPL], vr[GG][CPL];
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const int e = clamp_id(readlane_i32(ev, s0 + i - sb), a.N);
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      ur[i][q] = cv[q] ? U[(int64_t)e * rc + l + kWave * q] : make_uint4(0, 0, 0, 0);
      vr[i][q] = cv[q] ? V[(int64_t)e * rc + l + kWave * q] : make_uint4(0, 0, 0, 0);
    }
  }
  // every row of the group is requested before the first product
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const int64_t p = t * a.hk + s0 + i;
    const float g = readlane_f32(gv, s0 + i - sb);
    float hs = 0.0f, ds = 0.0f;
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) {
        hs = fmaf(chunk_elem<BF16>(xr[q], k), chunk_elem<BF16>(ur[i][q], k), hs);
        ds = fmaf(dyr[q][k], chunk_elem<BF16>(vr[i][q], k), ds);
      }
    const float h = wave_sum_uniform(hs);
    const float da = wave_sum_uniform(ds);
    const float act = activation(a.act, h);
    const float dh = da * g * activation_grad(a.act, h);
    if (l == 0) {
      a.a[p] = g * act;
      a.dh[p] = dh;
      a.dgates[p] = da * act;
    }
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = fmaf(dh, chunk_elem<BF16>(ur[i][q], k), acc[q][k]);
  }
}

// Token pass: one wave per token. The token's experts and gates are read 64 slots at a time
// (one load per lane), and the slots then go through G at a time with all of their u and v
// rows in flight, whole groups first and the rest singly, so that no row load waits behind the
// previous slot's work. FULL: the row is exactly CPL * 64 chunks (no load carries a guard).
template <int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(256) void bwd_token_kernel(BwdArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int G = CPL >= 8 ? 1 : (CPL >= 4 ? 2 : 4);
  const int l = lane_id();
  const uint4* X = (const uint4*)a.x;
  const int64_t rc = a.nchunks;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = FULL || (l + kWave * q) < a.nchunks;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < a.T; t += stride) {
    uint4 xr[CPL];
    float dyr[CPL][EPC];
    float acc[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      const int c = l + kWave * q;
      xr[q] = cv[q] ? X[t * rc + c] : make_uint4(0, 0, 0, 0);
      const float4* dyc = (const float4*)(a.dy + t * a.d + (int64_t)c * EPC);
#pragma unroll
      for (int k = 0; k < EPC; k += 4) {
        const float4 y4 = cv[q] ? dyc[k / 4] : make_float4(0.f, 0.f, 0.f, 0.f);
        dyr[q][k] = y4.x;
        dyr[q][k + 1] = y4.y;
        dyr[q][k + 2] = y4.z;
        dyr[q][k + 3] = y4.w;
      }
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = 0.0f;
    }
    for (int sb = 0; sb < a.hk; sb += kWave) {
      const int n = a.hk - sb < kWave ? a.hk - sb : kWave;
      const int64_t pl = t * a.hk + sb + (l < n ? l : n - 1);
      const int ev = a.idx[pl];
      const float gv = a.gates[pl];
      int s0 = sb;
      for (; s0 + G <= sb + n; s0 += G)
        token_slots<G, CPL, BF16>(a, t, s0, sb, ev, gv, xr, dyr, cv, acc);
      for (; s0 < sb + n; ++s0) token_slots<1, CPL, BF16>(a, t, s0, sb, ev, gv, xr, dyr, cv, acc);
    }
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!cv[q]) continue;
      const int c = l + kWave * q;
      float4* o = (float4*)(a.dx + t * a.d + (int64_t)c * EPC);
#pragma unroll
      for (int k = 0; k < EPC; k += 4) o[k / 4] = make_float4(acc[q][k], acc[q][k + 1], acc[q][k + 2], acc[q][k + 3]);
    }
  }
}

// Tasks j0 .. j0 + GG - 1 of the lanes' batch (slot pl, a_p apl, dh_p dhl on lane j): all their
// token and dy rows are loaded, then du += dh_p x_t and dv += a_p dy_t in task order.
template <int GG, int CPL, bool BF16>
__device__ __forceinline__ void task_group(const BwdArgs& a, const uint4* X, int64_t rc,
                                           const bool (&cv)[CPL], int pl, float apl, float dhl,
                                           int j0, float (&du)[CPL][BF16 ? 8 : 4],
                                           float (&dv)[CPL][BF16 ? 8 : 4]) {
  constexpr int EPC = BF16 ? 8 : 4;
  const int l = lane_id();
  uint4 xr[GG][CPL];
  float4 yr[GG][CPL][EPC / 4];
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const int64_t t = readlane_i32(pl, j0 + i) / a.hk;
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      const int c = l + kWave * q;
      xr[i][q] = cv[q] ? X[t * rc + c] : make_uint4(0, 0, 0, 0);
      const float4* dyc = (const float4*)(a.dy + t * a.d + (int64_t)c * EPC);
#pragma unroll
      for (int k = 0; k < EPC / 4; ++k) yr[i][q][k] = cv[q] ? dyc[k] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  // every load above is issued before the first product (left alone, the scheduler interleaves
  // them with the products and waits for each row in turn)
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const float ap = readlane_f32(apl, j0 + i), dhp = readlane_f32(dhl, j0 + i);
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
#pragma unroll
      for (int k = 0; k < EPC; k += 4) {
        const float4 yv = yr[i][q][k / 4];
        dv[q][k] = fmaf(ap, yv.x, dv[q][k]);
        dv[q][k + 1] = fmaf(ap, yv.y, dv[q][k + 1]);
        dv[q][k + 2] = fmaf(ap, yv.z, dv[q][k + 2]);
        dv[q][k + 3] = fmaf(ap, yv.w, dv[q][k + 3]);
      }
#pragma unroll
      for (int k = 0; k < EPC; ++k) du[q][k] = fmaf(dhp, chunk_elem<BF16>(xr[i][q], k), du[q][k]);
    }
  }
}

// Expert pass. The segment's tasks are taken 64 at a time: lane j loads the j-th one's slot,
// a and dh (one round trip for all of them), and the tasks then go through in order, G at a time
// with all of their token and dy rows in flight before the first product (the sums keep task
// order, so du and dv are the same as with one task at a time). FULL: the row is exactly CPL * 64
// chunks and no load carries a guard (guarded loads made the compiler wait for each chunk).
template <int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(256) void bwd_expert_kernel(BwdArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int G = CPL >= 8 ? 1 : 2;
  const int l = lane_id();
  const uint4* X = (const uint4*)a.x;
  const int64_t rc = a.nchunks;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = FULL || (l + kWave * q) < a.nchunks;
  const int64_t na = *a.n_active < a.cap ? *a.n_active : a.cap;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < na; r += stride) {
    float du[CPL][EPC], dv[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) du[q][k] = dv[q][k] = 0.0f;
    int64_t b = a.offsets[r], e = a.offsets[r + 1];
    b = b < 0 ? 0 : (b > a.M ? a.M : b);
    e = e < b ? b : (e > a.M ? a.M : e);
    for (int64_t base = b; base < e; base += kWave) {
      const int n = (int)(e - base < kWave ? e - base : kWave);
      const int pl = clamp_id(a.perm[base + (l < n ? l : n - 1)], a.M);
      const float apl = a.a[pl], dhl = a.dh[pl];
      // whole groups of G tasks, then the remaining ones singly: every product of a group is
      // unconditional, so the compiler cannot move a task's loads behind the previous task's work
      int j0 = 0;
      for (; j0 + G <= n; j0 += G) task_group<G, CPL, BF16>(a, X, rc, cv, pl, apl, dhl, j0, du, dv);
      for (; j0 < n; ++j0) task_group<1, CPL, BF16>(a, X, rc, cv, pl, apl, dhl, j0, du, dv);
    }
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!cv[q]) continue;
      const int c = l + kWave * q;
      float4* ou = (float4*)(a.du + r * a.d + (int64_t)c * EPC);
      float4* ov = (float4*)(a.dv + r * a.d + (int64_t)c * EPC);
#pragma unroll
      for (int k = 0; k < EPC; k += 4) {
        ou[k / 4] = make_float4(du[q][k], du[q][k + 1], du[q][k + 2], du[q][k + 3]);
        ov[k / 4] = make_float4(dv[q][k], dv[q][k + 1], dv[q][k + 2], dv[q][k + 3]);
      }
    }
  }
}

__global__ __launch_bounds__(256) void bwd_score_kernel(BwdArgs a) {
  const int l = lane_id();
  const int64_t rows = a.T * (a.hk / a.K);
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); row < rows; row += stride) {
    const int64_t base = row * a.K;
    float part = 0.0f;
    for (int k = l; k < a.K; k += kWave) part = fmaf(a.gates[base + k], a.dgates[base + k], part);
    const float sgd = wave_sum_f32(part);
    for (int k = l; k < a.K; k += kWave)
      a.dscores[base + k] = a.gates[base + k] * (a.dgates[base + k] - sgd);
  }
}

// Sub-key of every task for one half: key = h * n_half + (row or column of the expert id).
__global__ __launch_bounds__(256) void subkey_kernel(const int32_t* idx, int32_t* key, int64_t m,
                                                     int hk, int K, int nc, int n_half, int col,
                                                     int64_t n_experts) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= m) return;
  const int e = clamp_id(idx[p], n_experts);
  const int h = (int)((p % hk) / K);
  key[p] = h * n_half + (col ? e % nc : e / nc);
}

struct KeySumArgs {
  const void* x;
  const float* ds;
  const int32_t* perm;
  const int32_t* active;
  const int32_t* offsets;
  const int32_t* n_active;
  float* dk;         // [H * n_half, d_key]
  int64_t M;
  int64_t cap;
  int64_t n_keys;
  int d;             // row length of x
  int dkey;
  int c0;            // first x column of this half's query
  int hk;
  int nchunks;       // 16-byte chunks of a d_key slice
};

// Tasks j0 .. j0 + GG - 1 of a keysum batch (slot pl, weight wl on lane j): their x slices are
// loaded together, then acc += ds_p x_t in task order.
template <int GG, int CPL, bool BF16>
__device__ __forceinline__ void keysum_group(const KeySumArgs& a, const uint4* X, int64_t xrc,
                                             int64_t c0, const bool (&cv)[CPL], int pl, float wl,
                                             int j0, float (&acc)[CPL][BF16 ? 8 : 4]) {
  constexpr int EPC = BF16 ? 8 : 4;
  const int l = lane_id();
  uint4 xr[GG][CPL];
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const int64_t t = readlane_i32(pl, j0 + i) / a.hk;
#pragma unroll
    for (int q = 0; q < CPL; ++q)
      xr[i][q] = cv[q] ? X[t * xrc + c0 + l + kWave * q] : make_uint4(0, 0, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);  // all of the group's loads before its first product
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const float w = readlane_f32(wl, j0 + i);
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = fmaf(w, chunk_elem<BF16>(xr[i][q], k), acc[q][k]);
  }
}

// One wavefront per selected sub-key: dk[key] = sum over its tasks (task order) of ds_p x_t.
// The segment's tasks are taken 64 at a time (slot and ds with one load per lane), then eight
// (or, with wide rows, fewer) at a time with their x slices in flight together; whole groups
// first and the rest singly, so that every product of a group is unconditional.
template <int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(256) void keysum_kernel(KeySumArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int G = CPL >= 8 ? 2 : (CPL >= 4 ? 4 : 8);
  const int l = lane_id();
  const int64_t xrc = a.d / EPC;   // chunks per x row
  const int64_t c0 = a.c0 / EPC;
  const uint4* X = (const uint4*)a.x;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = FULL || (l + kWave * q) < a.nchunks;
  const int64_t na = *a.n_active < a.cap ? *a.n_active : a.cap;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < na; r += stride) {
    float acc[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = 0.0f;
    int64_t b = a.offsets[r], e = a.offsets[r + 1];
    b = b < 0 ? 0 : (b > a.M ? a.M : b);
    e = e < b ? b : (e > a.M ? a.M : e);
    for (int64_t base = b; base < e; base += kWave) {
      const int n = (int)(e - base < kWave ? e - base : kWave);
      const int pl = clamp_id(a.perm[base + (l < n ? l : n - 1)], a.M);
      const float wl = a.ds[pl];
      int j0 = 0;
      for (; j0 + G <= n; j0 += G) keysum_group<G, CPL, BF16>(a, X, xrc, c0, cv, pl, wl, j0, acc);
      for (; j0 < n; ++j0) keysum_group<1, CPL, BF16>(a, X, xrc, c0, cv, pl, wl, j0, acc);
    }
    const int key = clamp_id(a.active[r], a.n_keys);
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!cv[q]) continue;
      float4* o = (float4*)(a.dk + (int64_t)key * a.dkey + (int64_t)(l + kWave * q) * EPC);
#pragma unroll
      for (int k = 0; k < EPC; k += 4) o[k / 4] = make_float4(acc[q][k], acc[q][k + 1], acc[q][k + 2], acc[q][k + 3]);
    }
  }
}

struct RouteDxArgs {
  const void* kr;
  const void* kc;
  const int32_t* idx;
  const float* ds;
  float* dx;
  int64_t T;
  int64_t N;
  int d;
  int dkey;
  int c0;
  int hk;
  int K;
  int nr, nc;
  int nchunks;   // 16-byte chunks of a d_key row
};

// Slots s0 .. s0 + GG - 1 of token t (expert on lane s - sb of ev, weight of wv): both sub-key
// rows of each are loaded together, then ar += ds_p keys_row[h, i_p] and ac += ds_p
// keys_col[h, j_p] in slot order.
template <int GG, int CPL, bool BF16>
__device__ __forceinline__ void route_dx_group(const RouteDxArgs& a, const bool (&cv)[CPL], int s0,
                                               int sb, int ev, float wv,
                                               float (&ar)[CPL][BF16 ? 8 : 4],
                                               float (&ac)[CPL][BF16 ? 8 : 4]) {
  constexpr int EPC = BF16 ? 8 : 4;
  const int l = lane_id();
  const uint4* KR = (const uint4*)a.kr;
  const uint4* KC = (const uint4*)a.kc;
  const int64_t rc = a.nchunks;
  uint4 rr[GG][CPL], cr[GG][CPL];
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const int s = s0 + i;
    const int e = clamp_id(readlane_i32(ev, s - sb), a.N);
    const int h = s / a.K;
    const int64_t ri = (int64_t)h * a.nr + e / a.nc;
    const int64_t cj = (int64_t)h * a.nc + e % a.nc;
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      rr[i][q] = cv[q] ? KR[ri * rc + l + kWave * q] : make_uint4(0, 0, 0, 0);
      cr[i][q] = cv[q] ? KC[cj * rc + l + kWave * q] : make_uint4(0, 0, 0, 0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);  // all of the group's loads before its first product
#pragma unroll
  for (int i = 0; i < GG; ++i) {
    const float w = readlane_f32(wv, s0 + i - sb);
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) {
        ar[q][k] = fmaf(w, chunk_elem<BF16>(rr[i][q], k), ar[q][k]);
        ac[q][k] = fmaf(w, chunk_elem<BF16>(cr[i][q], k), ac[q][k]);
      }
  }
}

// dx_t[0 : d_key] += sum of ds_p keys_row[h, i_p]; dx_t[c0 : c0 + d_key] += sum of ds_p
// keys_col[h, j_p]; one wavefront per token, slots in order: experts and weights read 64 slots
// at a time, then groups of slots with all of their sub-key rows in flight.
template <int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(256) void route_dx_kernel(RouteDxArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int G = CPL >= 8 ? 1 : (CPL >= 4 ? 2 : 4);
  const int l = lane_id();
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = FULL || (l + kWave * q) < a.nchunks;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < a.T; t += stride) {
    float ar[CPL][EPC], ac[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) ar[q][k] = ac[q][k] = 0.0f;
    for (int sb = 0; sb < a.hk; sb += kWave) {
      const int n = a.hk - sb < kWave ? a.hk - sb : kWave;
      const int64_t pl = t * a.hk + sb + (l < n ? l : n - 1);
      const int ev = a.idx[pl];
      const float wv = a.ds[pl];
      int s0 = sb;
      for (; s0 + G <= sb + n; s0 += G) route_dx_group<G, CPL, BF16>(a, cv, s0, sb, ev, wv, ar, ac);
      for (; s0 < sb + n; ++s0) route_dx_group<1, CPL, BF16>(a, cv, s0, sb, ev, wv, ar, ac);
    }
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!cv[q]) continue;
      float* o1 = a.dx + t * a.d + (int64_t)(l + kWave * q) * EPC;
      float* o2 = a.dx + t * a.d + a.c0 + (int64_t)(l + kWave * q) * EPC;
      if (a.c0 == 0) {
#pragma unroll
        for (int k = 0; k < EPC; ++k) o1[k] += ar[q][k] + ac[q][k];
      } else {
#pragma unroll
        for (int k = 0; k < EPC; ++k) {
          o1[k] += ar[q][k];
          o2[k] += ac[q][k];
        }
      }
    }
  }
}

template <int CPL, bool BF16>
void launch_router_bwd_kernels(const KeySumArgs& kr, const KeySumArgs& kc, const RouteDxArgs& rd,
                               int pass, hipStream_t st) {
  if (pass < 2) {
    const KeySumArgs& a = pass == 0 ? kr : kc;
    int64_t blocks = (a.cap + 3) / 4;
    if (blocks > 65536) blocks = 65536;
    if (a.nchunks == CPL * kWave)
      hipLaunchKernelGGL((keysum_kernel<CPL, BF16, true>), dim3((unsigned)blocks), dim3(256), 0,
                         st, a);
    else
      hipLaunchKernelGGL((keysum_kernel<CPL, BF16, false>), dim3((unsigned)blocks), dim3(256), 0,
                         st, a);
  } else {
    int64_t blocks = (rd.T + 3) / 4;
    if (blocks > 16384) blocks = 16384;
    if (rd.nchunks == CPL * kWave)
      hipLaunchKernelGGL((route_dx_kernel<CPL, BF16, true>), dim3((unsigned)blocks), dim3(256), 0,
                         st, rd);
    else
      hipLaunchKernelGGL((route_dx_kernel<CPL, BF16, false>), dim3((unsigned)blocks), dim3(256),
                         0, st, rd);
  }
}

template <bool BF16>
hipError_t dispatch_router_bwd(int cpl, const KeySumArgs& kr, const KeySumArgs& kc,
                               const RouteDxArgs& rd, int pass, hipStream_t st) {
  switch (cpl) {
    case 1: launch_router_bwd_kernels<1, BF16>(kr, kc, rd, pass, st); break;
    case 2: launch_router_bwd_kernels<2, BF16>(kr, kc, rd, pass, st); break;
    case 4: launch_router_bwd_kernels<4, BF16>(kr, kc, rd, pass, st); break;
    case 8: launch_router_bwd_kernels<8, BF16>(kr, kc, rd, pass, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int cpl_of(int nchunks) {
  int c = 1;
  while (c * kWave < nchunks) c <<= 1;
  return c;
}

template <bool BF16>
hipError_t dispatch_bwd(int cpl, int64_t t_blocks, int64_t e_blocks, hipStream_t st,
                        const BwdArgs& a) {
#define OMNIMOE_BWD(C)                                                                    \
  case C:                                                                                 \
    if (a.nchunks == C * kWave)                                                           \
      hipLaunchKernelGGL((bwd_token_kernel<C, BF16, true>), dim3((unsigned)t_blocks),       \
                         dim3(256), 0, st, a);                                            \
    else                                                                                  \
      hipLaunchKernelGGL((bwd_token_kernel<C, BF16, false>), dim3((unsigned)t_blocks),      \
                         dim3(256), 0, st, a);                                            \
    if (a.nchunks == C * kWave)                                                           \
      hipLaunchKernelGGL((bwd_expert_kernel<C, BF16, true>), dim3((unsigned)e_blocks),      \
                         dim3(256), 0, st, a);                                            \
    else                                                                                  \
      hipLaunchKernelGGL((bwd_expert_kernel<C, BF16, false>), dim3((unsigned)e_blocks),     \
                         dim3(256), 0, st, a);                                            \
    break;
  switch (cpl) {
    OMNIMOE_BWD(1)
    OMNIMOE_BWD(2)
    OMNIMOE_BWD(4)
    OMNIMOE_BWD(8)
    default:
      return hipErrorInvalidValue;
  }
#undef OMNIMOE_BWD
  return hipGetLastError();
}

}  // namespace

size_t backward_ws_bytes(int64_t M) { return 2 * (((size_t)M * 4 + 255) & ~(size_t)255); }

hipError_t launch_expert_backward(const Shape& s, const void* x, const void* u, const void* v,
                                  const int32_t* idx, const float* gates, const int32_t* perm,
                                  const int32_t* offsets, const int32_t* n_active,
                                  const float* dy, float* dx, float* du, float* dv,
                                  float* dgates, float* dscores, void* ws, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  BwdArgs a;
  a.x = x;
  a.u = u;
  a.v = v;
  a.idx = idx;
  a.gates = gates;
  a.dy = dy;
  a.perm = perm;
  a.offsets = offsets;
  a.n_active = n_active;
  a.dx = dx;
  a.du = du;
  a.dv = dv;
  a.dgates = dgates;
  a.dscores = dscores;
  a.a = (float*)ws;
  a.dh = (float*)((char*)ws + (((size_t)s.M * 4 + 255) & ~(size_t)255));
  a.T = s.T;
  a.N = s.N;
  a.M = s.M;
  a.cap = s.M < s.N ? s.M : s.N;
  a.d = s.d;
  a.hk = s.hk;
  a.K = s.K;
  a.act = s.act;
  a.nchunks = s.bf16 ? s.d / 8 : s.d / 4;
  const int cpl = cpl_of(a.nchunks);
  int64_t tb = (s.T + 3) / 4;
  if (tb > 16384) tb = 16384;
  int64_t eb = (a.cap + 3) / 4;
  if (eb > 65536) eb = 65536;
  hipError_t e = s.bf16 ? dispatch_bwd<true>(cpl, tb, eb, st, a)
                        : dispatch_bwd<false>(cpl, tb, eb, st, a);
  if (e != hipSuccess) return e;
  int64_t sb = (s.rows + 3) / 4;
  if (sb > 16384) sb = 16384;
  hipLaunchKernelGGL(bwd_score_kernel, dim3((unsigned)sb), dim3(256), 0, st, a);
  return hipGetLastError();
}

size_t route_backward_ws_bytes(const Shape& s) {
  const int64_t nkeys = (int64_t)s.H * (s.nr > s.nc ? s.nr : s.nc);
  const int64_t cap = s.M < nkeys ? s.M : nkeys;
  auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
  return 2 * al((size_t)s.M * 4) + al((size_t)s.M * 4) + 2 * al((size_t)(cap + 1) * 4) + 256 +
         schedule_ws_bytes(s.M, nkeys);
}

hipError_t launch_route_backward(const Shape& s, const void* x, const void* keys_row,
                                 const void* keys_col, const int32_t* idx, const float* dscores,
                                 float* dx, float* dkeys_row, float* dkeys_col, void* ws,
                                 hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  auto al = [](size_t v) { return (v + 255) & ~(size_t)255; };
  const int64_t nkeys = (int64_t)s.H * (s.nr > s.nc ? s.nr : s.nc);
  const int64_t cap = s.M < nkeys ? s.M : nkeys;
  char* w = (char*)ws;
  int32_t* rkey = (int32_t*)w; w += al((size_t)s.M * 4);
  int32_t* ckey = (int32_t*)w; w += al((size_t)s.M * 4);
  int32_t* perm = (int32_t*)w; w += al((size_t)s.M * 4);
  int32_t* active = (int32_t*)w; w += al((size_t)(cap + 1) * 4);
  int32_t* offsets = (int32_t*)w; w += al((size_t)(cap + 1) * 4);
  int32_t* n_active = (int32_t*)w; w += 256;
  void* sws = w;
  const int64_t mb = (s.M + 255) / 256;
  hipLaunchKernelGGL(subkey_kernel, dim3((unsigned)mb), dim3(256), 0, st, idx, rkey, s.M, s.hk,
                     s.K, s.nc, s.nr, 0, s.N);
  hipLaunchKernelGGL(subkey_kernel, dim3((unsigned)mb), dim3(256), 0, st, idx, ckey, s.M, s.hk,
                     s.K, s.nc, s.nc, 1, s.N);
  hipError_t e = launch_fill_i32((int32_t*)dkeys_row, (int64_t)s.H * s.nr * s.dk, 0, st);
  if (e == hipSuccess) e = launch_fill_i32((int32_t*)dkeys_col, (int64_t)s.H * s.nc * s.dk, 0, st);
  if (e != hipSuccess) return e;
  const int epc = s.bf16 ? 8 : 4;
  const int nchunks = s.dk / epc;
  const int cpl = cpl_of(nchunks);
  KeySumArgs ka;
  ka.x = x;
  ka.ds = dscores;
  ka.perm = perm;
  ka.active = active;
  ka.offsets = offsets;
  ka.n_active = n_active;
  ka.M = s.M;
  ka.d = s.d;
  ka.dkey = s.dk;
  ka.hk = s.hk;
  ka.nchunks = nchunks;
  RouteDxArgs rd;
  rd.kr = keys_row;
  rd.kc = keys_col;
  rd.idx = idx;
  rd.ds = dscores;
  rd.dx = dx;
  rd.T = s.T;
  rd.N = s.N;
  rd.d = s.d;
  rd.dkey = s.dk;
  rd.c0 = s.col0;
  rd.hk = s.hk;
  rd.K = s.K;
  rd.nr = s.nr;
  rd.nc = s.nc;
  rd.nchunks = nchunks;
  for (int half = 0; half < 2; ++half) {
    // the tasks sorted by this half's sub-key, then one wavefront per selected sub-key
    Shape ss = s;
    ss.N = (int64_t)s.H * (half ? s.nc : s.nr);
    ss.B = 1;
    const int32_t* sk = nullptr;
    e = launch_schedule(ss, half ? ckey : rkey, perm, active, offsets, n_active, nullptr, sws, &sk,
                        st);
    if (e != hipSuccess) return e;
    ka.cap = s.M < ss.N ? s.M : ss.N;
    ka.n_keys = ss.N;
    ka.c0 = half ? s.col0 : 0;
    ka.dk = half ? dkeys_col : dkeys_row;
    e = s.bf16 ? dispatch_router_bwd<true>(cpl, ka, ka, rd, 0, st)
               : dispatch_router_bwd<false>(cpl, ka, ka, rd, 0, st);
    if (e != hipSuccess) return e;
  }
  return s.bf16 ? dispatch_router_bwd<true>(cpl, ka, ka, rd, 2, st)
                : dispatch_router_bwd<false>(cpl, ka, ka, rd, 2, st);
}

}  // namespace omnimoe
