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

// The candidate cells (a, b) with (a + 1)(b + 1) <= K for every K <= 64, row rank major, one
// list per K (the lists for K = 1 .. 64 hold 8104 cells): a constant table, so that no
// workgroup builds its list before the first row. With fewer than K rows (columns) in the grid,
// the cells with a >= Kr (b >= Kc) are skipped where the list is read.
constexpr int kCandK = 64;
constexpr int kCandCells = 8104;
struct CandTable {
  uint16_t cell[kCandCells];  // (a << 8) | b
  uint16_t first[kCandK + 2];  // list of K: cell[first[K] .. first[K + 1])
};
constexpr CandTable make_cand_table() {
  CandTable t{};
  int c = 0;
  t.first[0] = 0;
  for (int K = 1; K <= kCandK; ++K) {
    t.first[K] = (uint16_t)c;
    for (int a = 0; a < K; ++a)
      for (int b = 0; (a + 1) * (b + 1) <= K; ++b) t.cell[c++] = (uint16_t)((a << 8) | b);
  }
  t.first[kCandK + 1] = (uint16_t)c;
  return t;
}
static_assert(make_cand_table().first[kCandK + 1] == kCandCells, "candidate table size");
__constant__ CandTable kCand = make_cand_table();

struct SelectArgs {
  const float* hs;
  int32_t* idx;
  float* gates;
  int64_t rows;
  int nr, nc, K;
  // fused slot-order dot (select_kernel with DCPL > 0): a[row K + k] = g * act(x_t . u_e) for
  // each pick, bf16 rows of exactly DCPL * 64 16-byte chunks
  const void* x;
  const void* u;
  float* abuf;
  int64_t N;
  int H, act;
};

// ---------------------------------------------------------------- cross-lane exchange
// x[l ^ J] for one 32-bit word: DPP for J < 16; for 16 and 32 the lane-half swaps of gfx950
// (v_permlane16_swap / v_permlane32_swap of the word with itself leave x[l ^ J] in one of the
// two results, chosen by lane), so no exchange goes through LDS.
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
    // results: rows (0, 0, 2, 2) and rows (1, 1, 3, 3) of 16 lanes
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return (lane_id() & 16) ? r[0] : r[1];
  } else {
    static_assert(J == 32, "xor_lane: J is a power of two below 64");
    // results: lanes (0-31, 0-31) and lanes (32-63, 32-63)
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (lane_id() & 32) ? r[0] : r[1];
  }
}

// Sum over the wave by a butterfly of xor exchanges (32, 16, ..., 1); every lane receives the
// same value, as the two partners of each level add the same two partial sums.
__device__ __forceinline__ float wave_sum_xor(float v) {
  v += __uint_as_float(xor_lane<32>(__float_as_uint(v)));
  v += __uint_as_float(xor_lane<16>(__float_as_uint(v)));
  v += __uint_as_float(xor_lane<8>(__float_as_uint(v)));
  v += __uint_as_float(xor_lane<4>(__float_as_uint(v)));
  v += __uint_as_float(xor_lane<2>(__float_as_uint(v)));
  v += __uint_as_float(xor_lane<1>(__float_as_uint(v)));
  return v;
}

template <int J>
__device__ __forceinline__ uint64_t xor_lane64(uint64_t v) {
  return ((uint64_t)xor_lane<J>((uint32_t)(v >> 32)) << 32) | xor_lane<J>((uint32_t)v);
}

__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return a > b ? a : b; }

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

// For each of two halves, a threshold th with at least k lanes holding a value >= th, at most
// the k-th largest lane value: a bitwise search with ballots for the k-th largest value that
// leaves the lowest kLowBits bits at zero. Those bits only move th by less than 2^kLowBits
// ordered steps, so at most a few extra logits survive; the selection stays exact. Both halves'
// searches run in one loop (two independent chains, so their latencies overlap).
constexpr int kLowBits = 8;
__device__ __forceinline__ void kth_largest_lane2(uint32_t va, int ka, uint32_t vb, int kb,
                                                  uint32_t* tha, uint32_t* thb) {
  uint32_t ta = 0u, tb = 0u;
#pragma unroll
  for (int b = 31; b >= kLowBits; --b) {
    const uint32_t ca = ta | (1u << b), cb = tb | (1u << b);
    const int na = __popcll(__ballot(va >= ca));
    const int nb = __popcll(__ballot(vb >= cb));
    if (na >= ka) ta = ca;
    if (nb >= kb) tb = cb;
  }
  *tha = ta;
  *thb = tb;
}

// Logits of one half held in registers. VEC: lane l holds 16-byte chunks, element
// j = 256 (k / 4) + 4 l + k % 4 (needs n % 4 == 0 and 16-byte aligned rows); otherwise element
// j = l + 64 k. Positions past n hold garbage and are masked by index.
template <int R, bool VEC>
__device__ __forceinline__ int elem_index(int k) {
  return VEC ? 256 * (k >> 2) + 4 * lane_id() + (k & 3) : lane_id() + kWave * k;
}

// FULL: n == 64 R, every register position holds a logit (no masks by index).
template <int R, bool VEC, bool FULL>
__device__ __forceinline__ void load_half(const float* __restrict__ p, int n, float (&v)[R]) {
  if constexpr (VEC) {
#pragma unroll
    for (int c = 0; c < R / 4; ++c) {
      const int j0 = 256 * c + 4 * lane_id();
      // The logits are read once: non-temporal loads leave the caches to the later kernels.
      typedef float f32x4_t __attribute__((ext_vector_type(4)));
      f32x4_t t = {0.f, 0.f, 0.f, 0.f};
      if (FULL || j0 < n) t = __builtin_nontemporal_load((const f32x4_t*)(p + j0));
      v[4 * c] = t.x;
      v[4 * c + 1] = t.y;
      v[4 * c + 2] = t.z;
      v[4 * c + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int j = elem_index<R, VEC>(k);
      v[k] = (FULL || j < n) ? p[j] : 0.f;
    }
  }
}

// Order keys of one half's logits in registers and their lane maximum.
template <int R, bool VEC, bool FULL>
__device__ __forceinline__ uint32_t half_keys(const float (&v)[R], int n, uint32_t (&o)[R]) {
  uint32_t mx = 0u;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    // 0 sits below every finite value
    o[k] = (FULL || elem_index<R, VEC>(k) < n) ? ord_f32(v[k]) : 0u;
    mx = o[k] > mx ? o[k] : mx;
  }
  return mx;
}

// Writes the keys of one half's logits >= theta to buf[0, 32) and returns their number (those
// beyond 32 are not written). Register position by register position: a ballot gives the
// position's survivors, each writes at the running count plus the number of lower lanes that
// also survive (the sort that follows makes the slot order irrelevant).
template <int R, bool VEC>
__device__ __forceinline__ int half_survivors(const uint32_t (&o)[R], uint32_t theta,
                                              uint64_t* buf) {
  int total = 0;  // the same on every lane
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const bool sv = o[k] >= theta;
    const uint64_t m = __ballot(sv);
    const int pos = total + (int)__builtin_amdgcn_mbcnt_hi(
                                (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (sv && pos < 32) buf[pos] = logit_key(o[k], elem_index<R, VEC>(k));
    total += __popcll(m);
  }
  return total;
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

// DCPL > 0: after a row's picks and gates, the same wave forms their a[p] in slot order (the
// layer's dot where it forms no schedule): the token row once, then the u rows four at a time,
// each product summed exactly as slot_dot_kernel sums it, so a[p] is the same on both paths.
// This saves the dot's launch and its reads of idx and gates at a decode step.
template <int R, bool VEC, bool FULL, int DCPL = 0>
__global__ __launch_bounds__(256) void select_kernel(SelectArgs a) {
  __shared__ uint64_t lists[4][2][kWave];  // per wave: sorted row keys, sorted column keys
  __shared__ uint64_t stage[4][kWave];     // per wave: survivors, rows at 0, columns at 32
  const int K = a.K;
  const int kr = K < a.nr ? K : a.nr;
  const int kc = K < a.nc ? K : a.nc;
  const uint16_t* cand = kCand.cell + kCand.first[K];
  const int P = kCand.first[K + 1] - kCand.first[K];
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
    load_half<R, VEC, FULL>(a.hs + row * (int64_t)(a.nr + a.nc), a.nr, vr);
    load_half<R, VEC, FULL>(a.hs + row * (int64_t)(a.nr + a.nc) + a.nr, a.nc, vc);
  }
  for (; row < a.rows; row += stride) {
    const float* hr = a.hs + row * (int64_t)(a.nr + a.nc);
    float nr_[R], nc_[R];
    const int64_t nxt = row + stride;
    if (nxt < a.rows) {
      load_half<R, VEC, FULL>(a.hs + nxt * (int64_t)(a.nr + a.nc), a.nr, nr_);
      load_half<R, VEC, FULL>(a.hs + nxt * (int64_t)(a.nr + a.nc) + a.nr, a.nc, nc_);
    }
    uint32_t o_r[R], o_c[R], th_r, th_c;
    const uint32_t mx_r = half_keys<R, VEC, FULL>(vr, a.nr, o_r);
    const uint32_t mx_c = half_keys<R, VEC, FULL>(vc, a.nc, o_c);
    kth_largest_lane2(mx_r, kr, mx_c, kc, &th_r, &th_c);
    const int cr = half_survivors<R, VEC>(o_r, th_r, st);
    const int cc = half_survivors<R, VEC>(o_c, th_c, st + 32);
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
      const int cell = c < P ? cand[c] : 0;
      if (c < P && (cell >> 8) < kr && (cell & 0xFF) < kc) {
        const uint64_t kr_c = rowk[cell >> 8];
        const uint64_t kc_c = colk[cell & 0xFF];
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
    const double s0 = f64_from_ord(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(best.s >> 32), 0) << 32) |
                                   (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)best.s, 0));
    const float e = (l < K) ? expf((float)(s - s0)) : 0.0f;
    const float z = wave_sum_xor(e);
    if (l < K) {
      a.idx[row * K + l] = (int32_t)(0xFFFFFFFFu - best.nn);
      a.gates[row * K + l] = e / z;
    }
    if constexpr (DCPL > 0) {
      typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
      const uint4* X = (const uint4*)a.x + (row / a.H) * (int64_t)(DCPL * kWave);
      const uint4* U = (const uint4*)a.u;
      const int eid = (int)(0xFFFFFFFFu - best.nn);  // lane k < K: the k-th pick
      uint4 xr[DCPL];
#pragma unroll
      for (int q = 0; q < DCPL; ++q) xr[q] = X[l + kWave * q];
      float hv = 0.0f;
      for (int j0 = 0; j0 < K; j0 += 4) {
        uint4 ur[4][DCPL];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int ei = readlane_i32(eid, j0 + i < K ? j0 + i : K - 1);
          ei = ei < 0 ? 0 : (ei >= a.N ? (int)(a.N - 1) : ei);
          const u32x4_t* ub = (const u32x4_t*)(U + (int64_t)ei * (DCPL * kWave));
#pragma unroll
          for (int q = 0; q < DCPL; ++q) {
            const u32x4_t v = __builtin_nontemporal_load(ub + l + kWave * q);
            ur[i][q] = make_uint4(v.x, v.y, v.z, v.w);
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float acc = 0.0f;
#pragma unroll
          for (int q = 0; q < DCPL; ++q) acc = chunk_dot<true>(ur[i][q], xr[q], acc);
          const float hs = wave_sum_uniform(acc);
          if (l == j0 + i) hv = hs;
        }
      }
      if (l < K) a.abuf[row * K + l] = (e / z) * activation(a.act, hv);
    }
#pragma unroll
    for (int k = 0; k < R; ++k) {
      vr[k] = nr_[k];
      vc[k] = nc_[k];
    }
  }
}

// ---------------------------------------------------------------- large K (65 .. 4096)
// One workgroup per (token, head) row, for K beyond one wavefront (eight waves when the final
// order holds 2048 keys or more, four below, where more rows share a compute unit):
//   1. each half is put in (logit desc, index asc) order: a half of at most 512 logits by a
//      bitonic sort in one wave's registers (the two halves on two waves), a longer half by a
//      bitonic sort in LDS;
//   2. the K-th largest cell score s* of the grid of the top Kr rows and top Kc columns (the
//      whole top K lies in it, see the file header). Row rank a holds the cells (a, b) in
//      descending score as b grows, so the number of its cells scoring at least u is found by
//      a binary search over the sorted columns. An interval [lo, hi) of ordered-double keys
//      with count(>= lo) >= K > count(>= hi) is cut in four at every step (three counts per
//      step, each row searching only between its counts at the two ends), until one of the
//      counts is exactly K or the interval holds a single score;
//   3. when several cells score exactly s*, the ones with the lowest ids are taken: within a
//      row rank such cells have equal column logits, so their column indices ascend with b,
//      and a second interval search over the id finds the smallest id bound that admits K;
//   4. the selected cells of row rank a are then its first t_a columns: they are written out
//      at the offsets of an exclusive scan of t_a, one run per row rank, each run already in
//      the final order (score descending, id ascending);
//   5. from 1024 keys on the runs are merged pairwise, level by level (merge path, in place);
//      up to 512 keys a bitonic sort over LDS is faster;
//   6. gates: softmax over the K scores, summed in a fixed order.
// Scores are compared as exact doubles (sums of two floats), integer keys elsewhere, so the
// result is exact and independent of thread timing.

constexpr int kLargeMaxWaves = 8;  // workgroups of 256 or 512 threads
constexpr int kMergeMinKeys = 1024;  // final order by merging the runs from k2 = 1024 keys on

struct LargeArgs {
  const float* hs;
  int32_t* idx;
  float* gates;
  int64_t rows;
  int nr, nc, K;
  int n2;   // power of two >= max(nr, nc)
  int k2;   // power of two >= K
};

// LDS after the sorted halves: the selected keys (k2 of 12 bytes).
size_t large_region_bytes(int, int k2) { return (size_t)k2 * 12; }
__device__ __forceinline__ int large_region_bytes_dev(int, int k2) { return k2 * 12; }

// Bytes of dynamic LDS the kernel needs: the sorted halves, the key region, and two arrays of
// kr + 1 counts per row rank.
size_t large_lds_bytes(int n2, int k2, int kr) {
  return (size_t)2 * n2 * 8 + large_region_bytes(n2, k2) + (size_t)2 * (kr + 1) * 4;
}

struct LargeShared {
  int cnt[2][3][kLargeMaxWaves];  // per-wave partial counts, two buffers used in turn
  int wint[kLargeMaxWaves];
  float wsum[kLargeMaxWaves];
  uint64_t wmax[kLargeMaxWaves];
};

// Number of columns b in [lo, hi) of row value r (ascending b = descending column logit) whose
// cell scores at least u (ordered-double key); the answer is known to lie in [lo, hi].
__device__ __forceinline__ int cells_at_least(const uint64_t* ck, double r, uint64_t u, int lo,
                                              int hi) {
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    const double s = r + (double)f32_from_ord((uint32_t)(ck[mid] >> 32));
    if (ord_f64(s) >= u) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Number of columns b in [lo, hi) whose cell id i * nc + j (column index j = ~key low word)
// is at most x; j ascends with b inside a run of equal column logits, which [lo, hi) is.
__device__ __forceinline__ int ids_at_most(const uint64_t* ck, int64_t base, int64_t x, int lo,
                                           int hi) {
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    const int64_t id = base + (int64_t)(0xFFFFFFFFu - (uint32_t)ck[mid]);
    if (id <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Sum over the workgroup of three per-thread counts; every thread gets the totals. Buffer
// `buf` alternates between calls, so one barrier per call suffices: a buffer is written again
// only after the barrier of the next call, which every thread passes after reading it.
template <int NW>
__device__ __forceinline__ void block_sum3(LargeShared& sh, int (&v)[3], int w, int l, int buf) {
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const int t = wave_sum_uniform_i32(v[q]);
    if (l == 0) sh.cnt[buf][q][w] = t;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    int t = 0;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) t += sh.cnt[buf][q][ww];
    v[q] = t;
  }
}

// Descending bitonic sort of 512 keys held by one wave, eight consecutive keys per lane
// (key i = 8 lane + q in x[q]): partner distances below 8 are exchanges between a lane's own
// registers, larger ones swap with lane l ^ (distance / 8) through DPP and the lane-half swaps.
template <int J>
__device__ __forceinline__ void ce_lanes(uint64_t (&x)[8], int k) {
  const int l = lane_id();
  const bool lower = (l & J) == 0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const uint64_t o = xor_lane64<J>(x[q]);
    const bool desc = ((8 * l + q) & k) == 0;
    x[q] = (lower == desc) ? (x[q] > o ? x[q] : o) : (x[q] > o ? o : x[q]);
  }
}

__device__ __forceinline__ void wave_sort512_desc(uint64_t (&x)[8]) {
  const int l = lane_id();
#pragma unroll
  for (int lk = 1; lk <= 9; ++lk) {
    const int k = 1 << lk;
#pragma unroll
    for (int lj = lk - 1; lj >= 0; --lj) {
      const int j = 1 << lj;
      if (j >= 8) {
        switch (j >> 3) {
          case 1: ce_lanes<1>(x, k); break;
          case 2: ce_lanes<2>(x, k); break;
          case 4: ce_lanes<4>(x, k); break;
          case 8: ce_lanes<8>(x, k); break;
          case 16: ce_lanes<16>(x, k); break;
          default: ce_lanes<32>(x, k); break;
        }
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (q & j) continue;
          const bool desc = ((8 * l + q) & k) == 0;
          const uint64_t p0 = x[q], p1 = x[q + j];
          const bool swap = desc ? (p0 < p1) : (p0 > p1);
          x[q] = swap ? p1 : p0;
          x[q + j] = swap ? p0 : p1;
        }
      }
    }
  }
}

// RPT: row ranks per thread in the searches (kr <= RPT * NT). MERGE: the final order by merging
// the runs (k2 >= 1024), else by a bitonic sort (k2 <= 512, four waves).
template <int NT, int RPT, bool MERGE>
__global__ __launch_bounds__(NT, NT == 256 ? 5 : 4) void select_large_kernel(LargeArgs a) {
  constexpr int kRowsPerThread = RPT;
  constexpr int kLargeThreads = NT;
  constexpr int kLargeWaves = NT / kWave;
  static_assert(kLargeWaves <= kLargeMaxWaves, "workgroup size");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ LargeShared sh;
  const int n2 = a.n2, k2 = a.k2, K = a.K;
  const int kr = K < a.nr ? K : a.nr;
  const int kc = K < a.nc ? K : a.nc;
  uint64_t* hk = (uint64_t*)smem;                 // [2][n2]: rows, then columns
  uint64_t* sel_s = hk + 2 * n2;                  // [k2]
  uint32_t* sel_n = (uint32_t*)(sel_s + k2);      // [k2]
  // per row rank: the search brackets (counts at the interval's two ends), later t_a and the
  // exclusive scan of t_a
  int* cnt_lo = (int*)((unsigned char*)sel_s + large_region_bytes_dev(n2, k2));  // [kr + 1]
  int* cnt_hi = cnt_lo + (kr + 1);                                                 // [kr + 1]
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  const uint64_t* ck = hk + n2;

  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* hr = a.hs + row * (int64_t)(a.nr + a.nc);
    // 1. the top kr row keys and top kc column keys, descending. Halves of at most 512 logits:
    // wave 0 sorts the rows and wave 1 the columns, each in its registers; longer halves: a
    // bitonic sort in LDS by the whole workgroup. Keys are padded with 0 (below every finite
    // logit).
    if (n2 <= 512) {
      if (w < 2) {
        const int n = w == 0 ? a.nr : a.nc;
        const float* src = hr + (w == 0 ? 0 : a.nr);
        uint64_t x[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int j = 8 * l + q;
          x[q] = j < n ? logit_key(ord_f32(src[j]), j) : 0ull;
        }
        wave_sort512_desc(x);
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (8 * l + q < n2) hk[w * n2 + 8 * l + q] = x[q];
      }
      __syncthreads();
    } else {
      // keys padded with 0 (below every finite logit), both halves sorted descending
      for (int i = tid; i < 2 * n2; i += kLargeThreads) {
        const int h = i >= n2, j = i - h * n2;
        const int n = h ? a.nc : a.nr;
        hk[i] = j < n ? logit_key(ord_f32(hr[h * a.nr + j]), j) : 0ull;
      }
      __syncthreads();
      for (int lk = 1; (1 << lk) <= n2; ++lk) {
        const int k = 1 << lk;
        for (int lj = lk - 1; lj >= 0; --lj) {
          const int j = 1 << lj;
          for (int t = tid; t < n2; t += kLargeThreads) {
            const int i = ((t >> lj) << (lj + 1)) | (t & (j - 1));
            const uint64_t x = hk[i], y = hk[i + j];
            const bool up = (i & k & (n2 - 1)) == 0;
            if ((x < y) == up) {
              hk[i] = y;
              hk[i + j] = x;
            }
          }
          __syncthreads();
        }
      }
    }
    // 2. the K-th largest score. Start: hi above the largest score (row rank 0 + column rank 0);
    // lo the best corner bound, r[A - 1] + c[B - 1] over A x B blocks of the sorted grid with
    // A B >= K (each such block holds K cells at or above its last one). Only the Cartesian
    // candidates b < min(Kc, K / (a + 1)) are counted: every cell scoring above the K-th score
    // is one, and a cell past the bound can at most tie with it, behind K cells (file header),
    // so counting the candidates finds the same score and, below, the same tied cells.
    uint64_t lo = 0ull, hi;
    {
      const int amin = (K + kc - 1) / kc;
      for (int A = amin + tid; A <= kr; A += kLargeThreads) {
        const int Bn = (K + A - 1) / A;  // <= kc
        const double v = (double)f32_from_ord((uint32_t)(hk[A - 1] >> 32)) +
                         (double)f32_from_ord((uint32_t)(ck[Bn - 1] >> 32));
        const uint64_t o = ord_f64(v);
        lo = o > lo ? o : lo;
      }
      lo = max_u64(lo, xor_lane64<32>(lo));
      lo = max_u64(lo, xor_lane64<16>(lo));
      lo = max_u64(lo, xor_lane64<8>(lo));
      lo = max_u64(lo, xor_lane64<4>(lo));
      lo = max_u64(lo, xor_lane64<2>(lo));
      lo = max_u64(lo, xor_lane64<1>(lo));
      if (l == 0) sh.wmax[w] = lo;
      __syncthreads();
#pragma unroll
      for (int ww = 0; ww < kLargeWaves; ++ww) lo = sh.wmax[ww] > lo ? sh.wmax[ww] : lo;
      hi = ord_f64((double)f32_from_ord((uint32_t)(hk[0] >> 32)) +
                   (double)f32_from_ord((uint32_t)(ck[0] >> 32))) + 1ull;
    }
    // this thread's row ranks r = tid + i NT: value, and the bracket [count at hi, count at lo]
    double rv[kRowsPerThread];
    int b_hi[kRowsPerThread], b_lo[kRowsPerThread];
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
      const int r = tid + i * kLargeThreads;
      rv[i] = r < kr ? (double)f32_from_ord((uint32_t)(hk[r] >> 32)) : 0.0;
      b_hi[i] = 0;
      const int cap = K / (r + 1);
      b_lo[i] = r < kr ? (cap < kc ? cap : kc) : 0;
    }
    int buf = 0;
    bool done = false;
    while (hi - lo > 1ull) {  // lo and hi are the same on every thread
      const uint64_t step = (hi - lo) >> 2;
      uint64_t u[3];
#pragma unroll
      for (int q = 0; q < 3; ++q) {
        const uint64_t o = step ? step * (uint64_t)(q + 1) : (uint64_t)(q + 1);
        u[q] = lo + (o < hi - lo ? o : hi - lo - 1);
      }
      int cnt[kRowsPerThread][3];
      int tot[3] = {0, 0, 0};
#pragma unroll
      for (int i = 0; i < kRowsPerThread; ++i) {
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          cnt[i][q] = cells_at_least(ck, rv[i], u[q], b_hi[i], b_lo[i]);
          tot[q] += cnt[i][q];
        }
      }
      block_sum3<kLargeWaves>(sh, tot, w, l, buf);
      buf ^= 1;
      const int exact = tot[0] == K ? 0 : (tot[1] == K ? 1 : (tot[2] == K ? 2 : -1));
      if (exact >= 0) {  // the selection is the cells scoring at least u[exact]
#pragma unroll
        for (int i = 0; i < kRowsPerThread; ++i) b_lo[i] = cnt[i][exact];
        done = true;
        break;
      }
      // the piece [u_j, u_j+1) holding the K-th score, u_0 = lo and u_4 = hi
      int j = 0;
#pragma unroll
      for (int q = 0; q < 3; ++q) j += tot[q] >= K ? 1 : 0;
#pragma unroll
      for (int i = 0; i < kRowsPerThread; ++i) {
        if (j > 0) b_lo[i] = cnt[i][j - 1];
        if (j < 3) b_hi[i] = cnt[i][j];
      }
      if (j > 0) lo = u[j - 1];
      if (j < 3) hi = u[j];
    }
    // 3. unless a count hit K, the interval holds the one score s* = lo. b_hi counts the
    // candidates of a row above it and b_lo those at or above it (both ends were counted, or
    // are the start's bounds; the rows confirm them here).
    if (!done) {
      int tot[3] = {0, 0, 0};
#pragma unroll
      for (int i = 0; i < kRowsPerThread; ++i) {
        const int r = tid + i * kLargeThreads;
        const int cap = K / (r + 1);
        const int g = cells_at_least(ck, rv[i], hi, 0, r < kr ? (cap < kc ? cap : kc) : 0);
        const int e = cells_at_least(ck, rv[i], lo, g, r < kr ? (cap < kc ? cap : kc) : 0);
        b_hi[i] = g;
        b_lo[i] = e;
        tot[0] += g;
        tot[1] += e;
      }
      block_sum3<kLargeWaves>(sh, tot, w, l, buf);
      buf ^= 1;
      const int krem = K - tot[0];  // cells to take among those scoring exactly s*
      if (tot[1] - tot[0] > krem) {
        // the smallest id bound x with krem tied cells of id <= x; invariant
        // count(<= xlo) < krem <= count(<= xhi)
        int64_t xlo = -1, xhi = (int64_t)a.nr * a.nc - 1;
        // id of the row's first column: i a.nc, i the row index of rank r (read from LDS)
        auto base = [&](int i) -> int64_t {
          const int r = tid + i * kLargeThreads;
          return r < kr ? (int64_t)(0xFFFFFFFFu - (uint32_t)hk[r]) * a.nc : 0;
        };
        while (xhi - xlo > 1) {
          const int64_t step = (xhi - xlo) >> 2;
          int64_t xs[3];
#pragma unroll
          for (int q = 0; q < 3; ++q) {
            const int64_t o = step ? step * (q + 1) : (int64_t)(q + 1);
            xs[q] = xlo + (o < xhi - xlo ? o : xhi - xlo - 1);
          }
          int t3[3] = {0, 0, 0};
#pragma unroll
          for (int i = 0; i < kRowsPerThread; ++i)
#pragma unroll
            for (int q = 0; q < 3; ++q)
              t3[q] += ids_at_most(ck, base(i), xs[q], b_hi[i], b_lo[i]) - b_hi[i];
          block_sum3<kLargeWaves>(sh, t3, w, l, buf);
          buf ^= 1;
          int j = 0;  // thresholds that admit fewer than krem
#pragma unroll
          for (int q = 0; q < 3; ++q) j += t3[q] >= krem ? 0 : 1;
          if (j > 0) xlo = xs[j - 1];
          if (j < 3) xhi = xs[j];
        }
#pragma unroll
        for (int i = 0; i < kRowsPerThread; ++i)
          b_lo[i] = ids_at_most(ck, base(i), xhi, b_hi[i], b_lo[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
      const int r = tid + i * kLargeThreads;
      if (r < kr) cnt_lo[r] = b_lo[i];
    }
    __syncthreads();
    // 4. t_a = cnt_lo[a] selected cells in row rank a: exclusive scan into cnt_hi, then the
    // keys at their offsets. Threads scan contiguous chunks of row ranks.
    {
      const int per = (kr + kLargeThreads - 1) / kLargeThreads;
      const int a0 = tid * per;
      int loc = 0;
      for (int q = a0; q < a0 + per && q < kr; ++q) loc += cnt_lo[q];
      const int ex = wave_excl_scan_i32(loc);
      if (l == kWave - 1) sh.wint[w] = ex + loc;
      __syncthreads();
      int off = 0;
      for (int ww = 0; ww < w; ++ww) off += sh.wint[ww];
      int run = off + ex;
      for (int q = a0; q < a0 + per && q < kr; ++q) {
        cnt_hi[q] = run;
        run += cnt_lo[q];
      }
      if (a0 < kr && a0 + per >= kr) cnt_hi[kr] = run;  // = K
      __syncthreads();
      // each thread writes a contiguous chunk of positions: one search for the row rank of its
      // first position (the last rank whose offset is <= it), then a walk along the rows
      const int chunk = (K + kLargeThreads - 1) / kLargeThreads;
      const int q0 = tid * chunk;
      const int q1 = q0 + chunk < K ? q0 + chunk : K;
      if (q0 < q1) {
        int ra = 0, hi = kr - 1;
        while (ra < hi) {
          const int mid = (ra + hi + 1) >> 1;
          if (cnt_hi[mid] <= q0) ra = mid; else hi = mid - 1;
        }
        int next = cnt_hi[ra + 1];  // first position of the next row rank
        uint64_t rk = hk[ra];
        double rvv = (double)f32_from_ord((uint32_t)(rk >> 32));
        uint32_t rid = (0xFFFFFFFFu - (uint32_t)rk) * (uint32_t)a.nc;
        for (int q = q0; q < q1; ++q) {
          while (q >= next) {  // row ranks with no selected cell are skipped
            ++ra;
            next = cnt_hi[ra + 1];
            rk = hk[ra];
            rvv = (double)f32_from_ord((uint32_t)(rk >> 32));
            rid = (0xFFFFFFFFu - (uint32_t)rk) * (uint32_t)a.nc;
          }
          const uint64_t cq = ck[q - cnt_hi[ra]];
          sel_s[q] = ord_f64(rvv + (double)f32_from_ord((uint32_t)(cq >> 32)));
          sel_n[q] = 0xFFFFFFFFu - (rid + (0xFFFFFFFFu - (uint32_t)cq));
        }
      }
    }
    __syncthreads();
    // 5. the final order. Row rank a's selected cells are already in it (descending score,
    // ascending id: its columns are in descending logit order, equal logits by ascending
    // index), so the K keys are kr sorted runs at the offsets cnt_hi. They are merged pairwise,
    // level by level: at level L the runs of row ranks [2m 2^L, (2m + 1) 2^L) and
    // [(2m + 1) 2^L, (2m + 2) 2^L) become one. Each thread produces kOut consecutive outputs:
    // the split of its first output between the two inputs comes from a binary search along
    // the merge path, the rest from a sequential merge with the two heads in registers (moving
    // on to the next run where one ends); after a barrier the outputs are written in place.
    // Keys are unique (distinct ids), so the order is fully determined.
    if constexpr (!MERGE) {
      // short lists (k2 <= 512): a bitonic sort over LDS (keys past K padded with 0, below
      // every key) takes fewer cycles than the merge levels (at K = 512: 25k against 31k)
      for (int i = K + tid; i < k2; i += kLargeThreads) {
        sel_s[i] = 0ull;
        sel_n[i] = 0u;
      }
      __syncthreads();
      for (int lk = 1; (1 << lk) <= k2; ++lk) {
        const int k = 1 << lk;
        for (int lj = lk - 1; lj >= 0; --lj) {
          const int j = 1 << lj;
          for (int t = tid; t < (k2 >> 1); t += kLargeThreads) {
            const int i = ((t >> lj) << (lj + 1)) | (t & (j - 1));
            const uint64_t xs = sel_s[i], ys = sel_s[i + j];
            const uint32_t xn = sel_n[i], yn = sel_n[i + j];
            const bool up = (i & k) == 0;
            const bool lt = xs < ys || (xs == ys && xn < yn);
            if (lt == up) {
              sel_s[i] = ys;
              sel_s[i + j] = xs;
              sel_n[i] = yn;
              sel_n[i + j] = xn;
            }
          }
          __syncthreads();
        }
      }
    } else {
      constexpr int kOut = NT == 512 ? 8 : 4;  // NT kOut >= k2 >= K
      const int o0 = tid * kOut;
      const int nout = o0 < K ? (K - o0 < kOut ? K - o0 : kOut) : 0;
      int a0 = 0;  // row rank holding position o0: the last a with cnt_hi[a] <= o0
      if (nout > 0) {
        int ahi = kr - 1;
        while (a0 < ahi) {
          const int mid = (a0 + ahi + 1) >> 1;
          if (cnt_hi[mid] <= o0) a0 = mid; else ahi = mid - 1;
        }
      }
      auto before = [](uint64_t s0, uint32_t n0, uint64_t s1, uint32_t n1) {
        return s0 > s1 || (s0 == s1 && n0 > n1);
      };
      for (int L = 0; (1 << L) < kr; ++L) {
        uint64_t os[kOut];
        uint32_t on[kOut];
        if (nout > 0) {
          // the merged run holding o0 (it holds row rank a0) and its inputs A = [as, ae),
          // B = [ae, be)
          int m = a0 >> (L + 1);
          const int as = cnt_hi[m << (L + 1)];
          int ae = cnt_hi[min((m << (L + 1)) + (1 << L), kr)];
          int be = cnt_hi[min((m + 1) << (L + 1), kr)];
          // merge path: the run's first d = o0 - as outputs are i keys of A and d - i of B
          const int d = o0 - as;
          int lo2 = d - (be - ae) > 0 ? d - (be - ae) : 0;
          int hi2 = d < ae - as ? d : ae - as;
          while (lo2 < hi2) {
            const int mid = (lo2 + hi2) >> 1;
            const int bj = ae + d - mid - 1;
            const uint64_t sa = sel_s[as + mid], sb = sel_s[bj];
            bool bf = sa > sb;
            if (sa == sb) bf = sel_n[as + mid] > sel_n[bj];  // ids only on equal scores
            if (bf) lo2 = mid + 1;
            else hi2 = mid;
          }
          int ia = as + lo2, ib = ae + d - lo2;
          // heads (key 0 past an input's end: below every key)
          uint64_t ha = ia < ae ? sel_s[ia] : 0ull, hb = ib < be ? sel_s[ib] : 0ull;
          uint32_t na = ia < ae ? sel_n[ia] : 0u, nb = ib < be ? sel_n[ib] : 0u;
#pragma unroll
          for (int q = 0; q < kOut; ++q) {
            if (q < nout) {
              const int o = o0 + q;
              if (o == be) {  // this run is done: the next nonempty one starts at o
                do {
                  ++m;
                  ae = cnt_hi[min((m << (L + 1)) + (1 << L), kr)];
                  be = cnt_hi[min((m + 1) << (L + 1), kr)];
                } while (be <= o);
                ia = o;
                ib = ae;
                ha = ia < ae ? sel_s[ia] : 0ull;
                na = ia < ae ? sel_n[ia] : 0u;
                hb = ib < be ? sel_s[ib] : 0ull;
                nb = ib < be ? sel_n[ib] : 0u;
              }
              const bool ta = before(ha, na, hb, nb);
              os[q] = ta ? ha : hb;
              on[q] = ta ? na : nb;
              // one read for the new head of the input just taken from (index clamped, the
              // key replaced by 0 past that input's end)
              if (ta) ++ia; else ++ib;
              const int nx = ta ? ia : ib;
              const bool live = nx < (ta ? ae : be);
              const int rx = nx < K ? nx : K - 1;
              const uint64_t ks = live ? sel_s[rx] : 0ull;
              const uint32_t kn = live ? sel_n[rx] : 0u;
              ha = ta ? ks : ha;
              na = ta ? kn : na;
              hb = ta ? hb : ks;
              nb = ta ? nb : kn;
            }
          }
        }
        __syncthreads();
        if (nout == kOut) {  // 16-byte stores (o0 is a multiple of kOut)
#pragma unroll
          for (int q = 0; q < kOut; q += 2)
            *(ulonglong2*)(sel_s + o0 + q) = make_ulonglong2(os[q], os[q + 1]);
#pragma unroll
          for (int q = 0; q < kOut; q += 4)
            *(uint4*)(sel_n + o0 + q) = make_uint4(on[q], on[q + 1], on[q + 2], on[q + 3]);
        } else {
#pragma unroll
          for (int q = 0; q < kOut; ++q) {
            if (q < nout) {
              sel_s[o0 + q] = os[q];
              sel_n[o0 + q] = on[q];
            }
          }
        }
        __syncthreads();
      }
    }
    // 6. gates: e_k = exp(S_k - S_0), summed per thread over a contiguous range, then across
    // lanes and waves in a fixed order
    const double s0 = f64_from_ord(sel_s[0]);
    const int per = (K + kLargeThreads - 1) / kLargeThreads;
    const int g0 = tid * per;
    float part = 0.0f;
    for (int q = g0; q < g0 + per && q < K; ++q)
      part += expf((float)(f64_from_ord(sel_s[q]) - s0));
    part = wave_sum_xor(part);
    if (l == 0) sh.wsum[w] = part;
    __syncthreads();
    float z = sh.wsum[0];
#pragma unroll
    for (int ww = 1; ww < kLargeWaves; ++ww) z += sh.wsum[ww];
    for (int q = tid; q < K; q += kLargeThreads) {
      a.idx[row * K + q] = (int32_t)(0xFFFFFFFFu - sel_n[q]);
      a.gates[row * K + q] = expf((float)(f64_from_ord(sel_s[q]) - s0)) / z;
    }
    __syncthreads();
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
      const float z = wave_sum_xor(e);
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
  if (s.K > kWave) {
    LargeArgs a;
    a.hs = half_scores;
    a.idx = idx;
    a.gates = gates;
    a.rows = s.rows;
    a.nr = s.nr;
    a.nc = s.nc;
    a.K = s.K;
    int n2 = 2;
    while (n2 < s.nr || n2 < s.nc) n2 <<= 1;
    int k2 = 2;
    while (k2 < s.K) k2 <<= 1;
    a.n2 = n2;
    a.k2 = k2;
    const int kr = s.K < s.nr ? s.K : s.nr;
    const size_t lds = large_lds_bytes(n2, k2, kr);
    const dim3 grid((unsigned)(s.rows < 4096 ? s.rows : 4096));
    // eight waves per row once the final order holds 2048 keys or more; four below, where
    // more rows share a compute unit. The final order comes from merging the runs from 1024
    // keys on, from a bitonic sort below. Each thread searches over ceil(kr / threads) row
    // ranks, rounded up to a power of two (kr <= K <= 4096).
    const int nt = k2 >= 2048 ? 512 : 256;
    const bool merge = k2 >= kMergeMinKeys;
    const int need = (kr + nt - 1) / nt;
    const int rpt = need <= 1 ? 1 : (need <= 2 ? 2 : (need <= 4 ? 4 : 8));
#define OMNIMOE_SELECT_LARGE(NT_, RPT_, M_)                                                \
  hipLaunchKernelGGL((select_large_kernel<NT_, RPT_, M_>), grid, dim3(NT_), lds, st, a)
    if (nt == 512) {
      if (rpt == 1) OMNIMOE_SELECT_LARGE(512, 1, true);
      else if (rpt == 2) OMNIMOE_SELECT_LARGE(512, 2, true);
      else if (rpt == 4) OMNIMOE_SELECT_LARGE(512, 4, true);
      else OMNIMOE_SELECT_LARGE(512, 8, true);
    } else if (merge) {
      if (rpt == 1) OMNIMOE_SELECT_LARGE(256, 1, true);
      else if (rpt == 2) OMNIMOE_SELECT_LARGE(256, 2, true);
      else OMNIMOE_SELECT_LARGE(256, 4, true);
    } else {
      if (rpt == 1) OMNIMOE_SELECT_LARGE(256, 1, false);
      else if (rpt == 2) OMNIMOE_SELECT_LARGE(256, 2, false);
      else OMNIMOE_SELECT_LARGE(256, 4, false);
    }
#undef OMNIMOE_SELECT_LARGE
    return hipGetLastError();
  }
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
    if (vec && (R) >= 4 && s.nr == 64 * (R) && s.nc == 64 * (R))                       \
      hipLaunchKernelGGL((select_kernel<(R), true, true>), grid, block, 0, st, a);     \
    else if (vec && (R) >= 4)                                                          \
      hipLaunchKernelGGL((select_kernel<(R), true, false>), grid, block, 0, st, a);    \
    else                                                                               \
      hipLaunchKernelGGL((select_kernel<(R), false, false>), grid, block, 0, st, a);   \
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

bool select_dot_fusable(const Shape& s) {
  const int nchunks = s.d / 8;
  const bool rows_ok = s.nr == s.nc && (s.nr == 256 || s.nr == 512 || s.nr == 1024);
  const bool dot_ok = nchunks == 64 || nchunks == 128 || nchunks == 256 || nchunks == 512;
  return s.bf16 && s.K <= kWave && s.d % 8 == 0 && rows_ok && dot_ok;
}

hipError_t launch_select_dot(const Shape& s, const float* half_scores, int32_t* idx,
                             float* gates, const void* x, const void* u, float* abuf,
                             hipStream_t st) {
  if (s.rows == 0) return hipSuccess;
  if (!select_dot_fusable(s)) return hipErrorNotSupported;
  SelectArgs a;
  a.hs = half_scores;
  a.idx = idx;
  a.gates = gates;
  a.rows = s.rows;
  a.nr = s.nr;
  a.nc = s.nc;
  a.K = s.K;
  a.x = x;
  a.u = u;
  a.abuf = abuf;
  a.N = s.N;
  a.H = s.H;
  a.act = s.act;
  int64_t blocks = (s.rows + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  const dim3 grid((unsigned)blocks), block(256);
  const int cpl = s.d / 8 / kWave;
#define OMNIMOE_SELECT_DOT(R_)                                                                 \
  do {                                                                                         \
    if (cpl == 1) hipLaunchKernelGGL((select_kernel<R_, true, true, 1>), grid, block, 0, st, a);      \
    else if (cpl == 2) hipLaunchKernelGGL((select_kernel<R_, true, true, 2>), grid, block, 0, st, a); \
    else if (cpl == 4) hipLaunchKernelGGL((select_kernel<R_, true, true, 4>), grid, block, 0, st, a); \
    else hipLaunchKernelGGL((select_kernel<R_, true, true, 8>), grid, block, 0, st, a);               \
  } while (0)
  if (s.nr == 256) OMNIMOE_SELECT_DOT(4);
  else if (s.nr == 512) OMNIMOE_SELECT_DOT(8);
  else OMNIMOE_SELECT_DOT(16);
#undef OMNIMOE_SELECT_DOT
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
