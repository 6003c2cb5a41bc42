// Router selection (Sec. 2.2, Eq. 11, 1, 2): for each (token, head) row of fp32 logits,
//   1. the top Kr = min(K, n_rows) rows and top Kc = min(K, n_cols) columns, each ranked by
//      (logit descending, index ascending);
//   2. the grid cells (a, b) of rank with (a + 1)(b + 1) <= K, scored S = s_r + s_c in double
//      (exact for two floats); every cell of the top K of the full grid is among them, since
//      a cell is preceded by all cells whose row and column ranks are both no worse;
//   3. the top K of those cells by (S descending, id ascending) and softmax gates over S.
// One wavefront per row. Keys are compared as integers (order-preserving bit maps), so the
// result is exact and independent of evaluation order.
//
// Per-half top-K: each lane holds ceil(n / 64) logits. theta, at most the Kh-th largest of
// the 64 lane maxima, is found by a bitwise search with ballots (Kh distinct lanes hold a
// value >= theta, so theta is at most the Kh-th largest logit and the logits >= theta contain
// the answer). Usually only a few more than Kh logits qualify: the two halves' survivors are
// compacted into lanes 0-31 (rows) and 32-63 (columns) and bitonic-sorted together. When more
// than 32 qualify (heavy ties, or K > 32) that half is instead sorted in batches of 64 from
// memory and merged.
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

constexpr int kMaxCand = 320;  // cells with (a+1)(b+1) <= 64: 280

struct SelectArgs {
  const float* hs;
  int32_t* idx;
  float* gates;
  int64_t rows;
  int nr, nc, K;
};

// ---------------------------------------------------------------- cross-lane exchange
// x[l ^ J] for one 32-bit word: DPP for J < 16, ds_swizzle for 16, ds_bpermute for 32.
template <int J>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v) {
  const int x = (int)v;
  if constexpr (J == 1) {
    return (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false);  // quad [1,0,3,2]
  } else if constexpr (J == 2) {
    return (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false);  // quad [2,3,0,1]
  } else if constexpr (J == 4) {
    const int lo = __builtin_amdgcn_update_dpp(x, x, 0x12C, 0xF, 0xF, false);  // row_ror:12
    const int hi = __builtin_amdgcn_update_dpp(x, x, 0x124, 0xF, 0xF, false);  // row_ror:4
    return (uint32_t)((lane_id() & 4) ? hi : lo);
  } else if constexpr (J == 8) {
    return (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x128, 0xF, 0xF, false);  // row_ror:8
  } else if constexpr (J == 16) {
    return (uint32_t)__builtin_amdgcn_ds_swizzle(x, (16 << 10) | 0x1F);  // bitmask xor 16
  } else {
    return (uint32_t)__shfl_xor(x, J, kWave);
  }
}

template <int J>
__device__ __forceinline__ uint64_t xor_lane64(uint64_t v) {
  return ((uint64_t)xor_lane<J>((uint32_t)(v >> 32)) << 32) | xor_lane<J>((uint32_t)v);
}

// 96-bit key of a grid cell: score (order map of the double) then lower id first.
struct CellKey {
  uint64_t s;
  uint32_t nn;  // ~id, so larger is better
};

__device__ __forceinline__ bool cell_gt(const CellKey& a, const CellKey& b) {
  return a.s > b.s || (a.s == b.s && a.nn > b.nn);
}

template <int J>
__device__ __forceinline__ CellKey xor_cell(const CellKey& k) {
  return CellKey{xor_lane64<J>(k.s), xor_lane<J>(k.nn)};
}

// One compare-exchange stage of a descending bitonic sort of segments of S lanes.
template <int S, int K2, int J>
__device__ __forceinline__ uint64_t stage64(uint64_t v) {
  const int l = lane_id();
  const uint64_t o = xor_lane64<J>(v);
  const bool up = (K2 >= S) ? true : ((l & K2) == 0);
  const bool keep_max = ((l & J) == 0) == up;
  const uint64_t mx = v > o ? v : o, mn = v > o ? o : v;
  return keep_max ? mx : mn;
}

template <int S, int K2, int J>
__device__ __forceinline__ CellKey stage_cell(CellKey v) {
  const int l = lane_id();
  const CellKey o = xor_cell<J>(v);
  const bool up = (K2 >= S) ? true : ((l & K2) == 0);
  const bool keep_max = ((l & J) == 0) == up;
  return (cell_gt(v, o) == keep_max) ? v : o;
}

// Descending bitonic sort within segments of S lanes (S = 32 or 64).
template <int S>
__device__ __forceinline__ uint64_t sort64(uint64_t v) {
  v = stage64<S, 2, 1>(v);
  v = stage64<S, 4, 2>(v); v = stage64<S, 4, 1>(v);
  v = stage64<S, 8, 4>(v); v = stage64<S, 8, 2>(v); v = stage64<S, 8, 1>(v);
  v = stage64<S, 16, 8>(v); v = stage64<S, 16, 4>(v); v = stage64<S, 16, 2>(v);
  v = stage64<S, 16, 1>(v);
  v = stage64<S, 32, 16>(v); v = stage64<S, 32, 8>(v); v = stage64<S, 32, 4>(v);
  v = stage64<S, 32, 2>(v); v = stage64<S, 32, 1>(v);
  if constexpr (S == 64) {
    v = stage64<S, 64, 32>(v); v = stage64<S, 64, 16>(v); v = stage64<S, 64, 8>(v);
    v = stage64<S, 64, 4>(v); v = stage64<S, 64, 2>(v); v = stage64<S, 64, 1>(v);
  }
  return v;
}

__device__ __forceinline__ CellKey sort_cells(CellKey v) {
  v = stage_cell<64, 2, 1>(v);
  v = stage_cell<64, 4, 2>(v); v = stage_cell<64, 4, 1>(v);
  v = stage_cell<64, 8, 4>(v); v = stage_cell<64, 8, 2>(v); v = stage_cell<64, 8, 1>(v);
  v = stage_cell<64, 16, 8>(v); v = stage_cell<64, 16, 4>(v); v = stage_cell<64, 16, 2>(v);
  v = stage_cell<64, 16, 1>(v);
  v = stage_cell<64, 32, 16>(v); v = stage_cell<64, 32, 8>(v); v = stage_cell<64, 32, 4>(v);
  v = stage_cell<64, 32, 2>(v); v = stage_cell<64, 32, 1>(v);
  v = stage_cell<64, 64, 32>(v); v = stage_cell<64, 64, 16>(v); v = stage_cell<64, 64, 8>(v);
  v = stage_cell<64, 64, 4>(v); v = stage_cell<64, 64, 2>(v); v = stage_cell<64, 64, 1>(v);
  return v;
}

// The final merge levels (segments of 64, already bitonic) of a descending sort.
__device__ __forceinline__ uint64_t bitonic_merge64(uint64_t v) {
  v = stage64<64, 64, 32>(v); v = stage64<64, 64, 16>(v); v = stage64<64, 64, 8>(v);
  v = stage64<64, 64, 4>(v); v = stage64<64, 64, 2>(v); v = stage64<64, 64, 1>(v);
  return v;
}
__device__ __forceinline__ CellKey bitonic_merge_cells(CellKey v) {
  v = stage_cell<64, 64, 32>(v); v = stage_cell<64, 64, 16>(v); v = stage_cell<64, 64, 8>(v);
  v = stage_cell<64, 64, 4>(v); v = stage_cell<64, 64, 2>(v); v = stage_cell<64, 64, 1>(v);
  return v;
}

// Top 64 of two descending lane-sorted lists, descending: lane l compares a[l] with
// b[63 - l] (the larger of each pair forms a bitonic sequence holding the top 64), then merges.
__device__ __forceinline__ uint64_t merge_top64(uint64_t a, uint64_t b) {
  const uint64_t rb = ((uint64_t)(uint32_t)__shfl((int)(b >> 32), (kWave - 1) - lane_id(), kWave) << 32) |
                      (uint32_t)__shfl((int)(uint32_t)b, (kWave - 1) - lane_id(), kWave);
  return bitonic_merge64(a > rb ? a : rb);
}
__device__ __forceinline__ CellKey merge_top64_cells(CellKey a, CellKey b) {
  const int src = (kWave - 1) - lane_id();
  CellKey rb;
  rb.s = ((uint64_t)(uint32_t)__shfl((int)(b.s >> 32), src, kWave) << 32) |
         (uint32_t)__shfl((int)(uint32_t)b.s, src, kWave);
  rb.nn = (uint32_t)__shfl((int)b.nn, src, kWave);
  return bitonic_merge_cells(cell_gt(a, rb) ? a : rb);
}

// ---------------------------------------------------------------- per-half top-K

// Key of logit j: value order in the high word, ~j in the low word (ties to lower j).
__device__ __forceinline__ uint64_t logit_key(uint32_t ord, int j) {
  return ((uint64_t)ord << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)j);
}

// A threshold th with at least k lanes holding a value >= th, at most the k-th largest lane
// value: a bitwise search with ballots for the k-th largest value that leaves the lowest
// kLowBits bits at zero. Those bits only move th by less than 2^kLowBits ordered steps, so at
// most a few extra logits survive; the selection stays exact.
constexpr int kLowBits = 8;
__device__ __forceinline__ uint32_t kth_largest_lane(uint32_t v, int k) {
  uint32_t th = 0u;
#pragma unroll
  for (int b = 31; b >= kLowBits; --b) {
    const uint32_t c = th | (1u << b);
    if (__popcll(__ballot(v >= c)) >= k) th = c;
  }
  return th;
}

// Logits of one half held in registers. VEC: lane l holds 16-byte chunks, element
// j = 256 (k / 4) + 4 l + k % 4 (needs n % 4 == 0 and 16-byte aligned rows); otherwise element
// j = l + 64 k. Positions past n hold garbage and are masked by index.
template <int R, bool VEC>
__device__ __forceinline__ int elem_index(int k) {
  return VEC ? 256 * (k >> 2) + 4 * lane_id() + (k & 3) : lane_id() + kWave * k;
}

template <int R, bool VEC>
__device__ __forceinline__ void load_half(const float* __restrict__ p, int n, float (&v)[R]) {
  if constexpr (VEC) {
#pragma unroll
    for (int c = 0; c < R / 4; ++c) {
      const int j0 = 256 * c + 4 * lane_id();
      float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
      if (j0 < n) t = *(const float4*)(p + j0);
      v[4 * c] = t.x;
      v[4 * c + 1] = t.y;
      v[4 * c + 2] = t.z;
      v[4 * c + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int j = elem_index<R, VEC>(k);
      v[k] = j < n ? p[j] : 0.f;
    }
  }
}

// Finds one half's threshold and writes the survivors' keys to buf[0, 32). Returns the number
// of survivors (those beyond 32 are not written).
template <int R, bool VEC>
__device__ __forceinline__ int half_survivors(const float (&v)[R], int n, int kh, uint64_t* buf,
                                              uint32_t* theta_out) {
  uint32_t o[R];
  uint32_t mx = 0u;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    o[k] = (elem_index<R, VEC>(k) < n) ? ord_f32(v[k]) : 0u;  // 0 sits below every finite value
    mx = o[k] > mx ? o[k] : mx;
  }
  const uint32_t theta = kth_largest_lane(mx, kh);
  *theta_out = theta;
  const uint64_t lt = lanemask_lt();
  int base = 0;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const bool f = o[k] >= theta;
    const uint64_t bal = __ballot(f);
    const int pos = base + __popcll(bal & lt);
    if (f && pos < 32) buf[pos] = logit_key(o[k], elem_index<R, VEC>(k));
    base += __popcll(bal);
  }
  return base;
}

// Slow path for one half: the logits >= theta, sorted in batches of 64 read from memory and
// merged; lane l < 64 ends with the l-th best key.
__device__ __noinline__ uint64_t half_topk_batched(const float* __restrict__ p, int n,
                                                   uint32_t theta) {
  const int l = lane_id();
  uint64_t best = 0ull;
  bool first = true;
  for (int base = 0; base < n; base += kWave) {
    const int j = base + l;
    uint64_t key = 0ull;
    if (j < n) {
      const uint32_t o = ord_f32(p[j]);
      if (o >= theta) key = logit_key(o, j);
    }
    if (__ballot(key != 0ull) == 0ull) continue;
    key = sort64<64>(key);
    best = first ? key : merge_top64(best, key);
    first = false;
  }
  return best;
}

template <int R, bool VEC>
__global__ __launch_bounds__(256) void select_kernel(SelectArgs a) {
  __shared__ uint16_t cand[kMaxCand];  // (a << 8) | b
  __shared__ int n_cand;
  __shared__ uint64_t lists[4][2][kWave];  // per wave: sorted row keys, sorted column keys
  __shared__ uint64_t stage[4][kWave];     // per wave: survivors, rows at 0, columns at 32
  const int K = a.K;
  const int kr = K < a.nr ? K : a.nr;
  const int kc = K < a.nc ? K : a.nc;
  if (threadIdx.x == 0) {
    int c = 0;
    for (int ra = 0; ra < kr; ++ra)
      for (int rb = 0; rb < kc && (ra + 1) * (rb + 1) <= K; ++rb)
        cand[c++] = (uint16_t)((ra << 8) | rb);
    n_cand = c;
  }
  __syncthreads();
  const int P = n_cand;
  const int l = lane_id();
  const int w = threadIdx.x >> 6;
  uint64_t* rowk = lists[w][0];
  uint64_t* colk = lists[w][1];
  uint64_t* st = stage[w];
  const int64_t stride = (int64_t)gridDim.x * 4;
  int64_t row = (int64_t)blockIdx.x * 4 + w;
  // The next row's logits are loaded while the current row is processed.
  float vr[R], vc[R];
  if (row < a.rows) {
    load_half<R, VEC>(a.hs + row * (int64_t)(a.nr + a.nc), a.nr, vr);
    load_half<R, VEC>(a.hs + row * (int64_t)(a.nr + a.nc) + a.nr, a.nc, vc);
  }
  for (; row < a.rows; row += stride) {
    const float* hr = a.hs + row * (int64_t)(a.nr + a.nc);
    float nr_[R], nc_[R];
    const int64_t nxt = row + stride;
    if (nxt < a.rows) {
      load_half<R, VEC>(a.hs + nxt * (int64_t)(a.nr + a.nc), a.nr, nr_);
      load_half<R, VEC>(a.hs + nxt * (int64_t)(a.nr + a.nc) + a.nr, a.nc, nc_);
    }
    uint32_t th_r, th_c;
    const int cr = half_survivors<R, VEC>(vr, a.nr, kr, st, &th_r);
    const int cc = half_survivors<R, VEC>(vc, a.nc, kc, st + 32, &th_c);
    wave_lds_sync();
    if (cr <= 32 && cc <= 32) {
      // Both halves in one pass: rows sort in lanes 0-31, columns in lanes 32-63.
      const int cnt = l < 32 ? cr : cc;
      uint64_t key = ((l & 31) < cnt) ? st[l] : 0ull;
      key = sort64<32>(key);
      if (l < 32) rowk[l] = key; else colk[l - 32] = key;
    } else {
      const uint64_t rk = cr <= 32 ? 0ull : half_topk_batched(hr, a.nr, th_r);
      const uint64_t ck = cc <= 32 ? 0ull : half_topk_batched(hr + a.nr, a.nc, th_c);
      uint64_t rs = 0ull, cs = 0ull;
      if (cr <= 32) rs = sort64<32>((l < 32 && l < cr) ? st[l] : 0ull);
      if (cc <= 32) cs = sort64<32>((l < 32 && l < cc) ? st[32 + l] : 0ull);
      rowk[l] = cr <= 32 ? rs : rk;
      colk[l] = cc <= 32 ? cs : ck;
    }
    wave_lds_sync();
    // Cartesian candidates, 64 per batch.
    CellKey best{0ull, 0u};
    for (int base = 0; base < P; base += kWave) {
      const int c = base + l;
      CellKey key{0ull, 0u};
      if (c < P) {
        const uint64_t kr_c = rowk[cand[c] >> 8];
        const uint64_t kc_c = colk[cand[c] & 0xFF];
        const float vr = f32_from_ord((uint32_t)(kr_c >> 32));
        const float vc = f32_from_ord((uint32_t)(kc_c >> 32));
        const uint32_t i = 0xFFFFFFFFu - (uint32_t)kr_c;
        const uint32_t j = 0xFFFFFFFFu - (uint32_t)kc_c;
        key.s = ord_f64((double)vr + (double)vc);
        key.nn = 0xFFFFFFFFu - (i * (uint32_t)a.nc + j);
      }
      key = sort_cells(key);
      best = (base == 0) ? key : merge_top64_cells(best, key);
    }
    wave_lds_sync();
    // Gates: softmax over the K selected scores, best first.
    const double s = f64_from_ord(best.s);
    const double s0 = __shfl(s, 0, kWave);
    const float e = (l < K) ? expf((float)(s - s0)) : 0.0f;
    const float z = wave_sum_f32(e);
    if (l < K) {
      a.idx[row * K + l] = (int32_t)(0xFFFFFFFFu - best.nn);
      a.gates[row * K + l] = e / z;
    }
#pragma unroll
    for (int k = 0; k < R; ++k) {
      vr[k] = nr_[k];
      vc[k] = nc_[k];
    }
  }
}

// ---------------------------------------------------------------- dense router (ablation)
// Top K of all N logits of one (token, head) row by (logit desc, id asc), then softmax gates:
// the router without the Cartesian product (Table 3). One workgroup of four waves per row.
//   1. every thread keeps the largest of its logits (16-byte loads when N % 4 == 0);
//   2. theta = the K-th largest of the 256 thread maxima (bitwise search with ballots), so at
//      least K logits are >= theta and the top K are among them;
//   3. each wave scans a quarter of the row 64 logits at a time; a batch holding logits >= theta
//      is bitonic-sorted and merged into the wave's running top 64;
//   4. wave 0 merges the four lists and writes ids and gates.
struct DenseArgs {
  const float* logits;
  int32_t* idx;
  float* gates;
  int64_t rows;
  int64_t N;
  int K;
};

__global__ __launch_bounds__(256) void select_dense_kernel(DenseArgs a) {
  __shared__ uint32_t tmax[256];
  __shared__ uint64_t lists[3][kWave];
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  const int64_t N = a.N;
  const int K = a.K;
  const bool vec = (N & 3) == 0;
  const int64_t quarter = (N + 3) / 4;
  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* p = a.logits + row * N;
    uint32_t mx = 0u;
    if (vec) {
      for (int64_t j = 4 * (int64_t)tid; j < N; j += 4 * 256) {
        const float4 f = *(const float4*)(p + j);
        const uint32_t m0 = max(ord_f32(f.x), ord_f32(f.y));
        const uint32_t m1 = max(ord_f32(f.z), ord_f32(f.w));
        mx = max(mx, max(m0, m1));
      }
    } else {
      for (int64_t j = tid; j < N; j += 256) mx = max(mx, ord_f32(p[j]));
    }
    tmax[tid] = mx;
    __syncthreads();
    uint32_t m4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) m4[i] = tmax[l + kWave * i];
    uint32_t th = 0u;
    for (int b = 31; b >= 0; --b) {
      const uint32_t c = th | (1u << b);
      int cnt = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) cnt += __popcll(__ballot(m4[i] >= c));
      if (cnt >= K) th = c;
    }
    const int64_t q0 = w * quarter;
    const int64_t q1 = q0 + quarter < N ? q0 + quarter : N;
    uint64_t best = 0ull;
    bool first = true;
    for (int64_t base = q0; base < q1; base += kWave) {
      const int64_t j = base + l;
      uint64_t key = 0ull;
      if (j < q1) {
        const uint32_t o = ord_f32(p[j]);
        if (o >= th) key = logit_key(o, (int)j);
      }
      if (__ballot(key != 0ull) == 0ull) continue;
      key = sort64<64>(key);
      best = first ? key : merge_top64(best, key);
      first = false;
    }
    if (w > 0) lists[w - 1][l] = best;
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < 3; ++i) best = merge_top64(best, lists[i][l]);
      const float v = f32_from_ord((uint32_t)(best >> 32));
      const float v0 = __shfl(v, 0, kWave);
      const float e = (l < K) ? expf(v - v0) : 0.0f;
      const float z = wave_sum_f32(e);
      if (l < K) {
        a.idx[row * K + l] = (int32_t)(0xFFFFFFFFu - (uint32_t)best);
        a.gates[row * K + l] = e / z;
      }
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_select(const Shape& s, const float* half_scores, int32_t* idx, float* gates,
                         hipStream_t st) {
  if (s.rows == 0) return hipSuccess;
  SelectArgs a;
  a.hs = half_scores;
  a.idx = idx;
  a.gates = gates;
  a.rows = s.rows;
  a.nr = s.nr;
  a.nc = s.nc;
  a.K = s.K;
  const int nmax = s.nr > s.nc ? s.nr : s.nc;
  int64_t blocks = (s.rows + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  dim3 grid((unsigned)blocks), block(256);
  const bool vec = s.nr % 4 == 0 && s.nc % 4 == 0;
#define OMNIMOE_SELECT(R)                                                              \
  do {                                                                                 \
    if (vec && (R) >= 4)                                                               \
      hipLaunchKernelGGL((select_kernel<(R), true>), grid, block, 0, st, a);           \
    else                                                                               \
      hipLaunchKernelGGL((select_kernel<(R), false>), grid, block, 0, st, a);          \
  } while (0)
  if (nmax <= 64) OMNIMOE_SELECT(1);
  else if (nmax <= 128) OMNIMOE_SELECT(2);
  else if (nmax <= 256) OMNIMOE_SELECT(4);
  else if (nmax <= 512) OMNIMOE_SELECT(8);
  else if (nmax <= 1024) OMNIMOE_SELECT(16);
  else if (nmax <= 2048) OMNIMOE_SELECT(32);
  else OMNIMOE_SELECT(64);
#undef OMNIMOE_SELECT
  return hipGetLastError();
}

hipError_t launch_select_dense(int64_t rows, int64_t n, int K, const float* logits, int32_t* idx,
                               float* gates, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  DenseArgs a;
  a.logits = logits;
  a.idx = idx;
  a.gates = gates;
  a.rows = rows;
  a.N = n;
  a.K = K;
  const dim3 grid((unsigned)(rows < 16384 ? rows : 16384));
  hipLaunchKernelGGL(select_dense_kernel, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace omnimoe
