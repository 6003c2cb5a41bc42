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

template <int R, bool VEC, bool FULL>
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
    const double s0 = f64_from_ord(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(best.s >> 32), 0) << 32) |
                                   (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)best.s, 0));
    const float e = (l < K) ? expf((float)(s - s0)) : 0.0f;
    const float z = wave_sum_xor(e);
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

// ---------------------------------------------------------------- large K (65 .. 4096)
// One workgroup per (token, head) row, for K beyond one wavefront (eight waves when the final
// sort holds 2048 keys or more, four below, where more rows share a compute unit):
//   1. each half is put in (logit desc, index asc) order. A half of at most 512 logits is
//      ordered by counting, for each key, the larger keys of its half (keys are distinct, so
//      that count is the key's rank); a longer half by a bitonic sort in LDS;
//   2. the Cartesian candidates (a, b) with (a+1)(b+1) <= K form a flat list (row rank a
//      holds min(Kc, floor(K / (a+1))) of them; the offsets depend only on (K, Kr, Kc) and are
//      computed once per workgroup), and each thread walks a contiguous chunk of it. A
//      candidate's key is (S as an order-preserving 64-bit integer, ~id);
//   3. a radix select over the 96-bit keys, eight bits at a time from the top (twelve passes
//      with an LDS histogram), finds the K-th largest key exactly. Passes walk every candidate
//      until the keys that share the decided prefix fit in LDS; the next pass also copies
//      those keys out, and the remaining passes read only the copy (one wave alone takes them
//      when the copy is short, with no workgroup barriers);
//   4. the K keys at or above the threshold are gathered and bitonic-sorted descending;
//   5. gates: softmax over the K scores, summed in a fixed order.
// Integer comparisons throughout, so the result is exact and independent of thread timing.

constexpr int kLargeMaxWaves = 8;  // workgroups of 256 or 512 threads
constexpr int kRankSortMax = 512;  // halves up to this padded length are ordered by counting
constexpr int kWaveFinish = 1024;  // radix survivors up to this many are finished by one wave

struct LargeArgs {
  const float* hs;
  int32_t* idx;
  float* gates;
  int64_t rows;
  int nr, nc, K;
  int n2;   // power of two >= max(nr, nc)
  int k2;   // power of two >= K
};

// LDS after the sorted halves: the selected keys (k2 of 12 bytes). Before the gather the
// same bytes hold the radix survivors and, when counting orders the halves, the unsorted
// half keys.
size_t large_region_bytes(int n2, int k2) {
  const size_t sel = (size_t)k2 * 12;
  const size_t stage = n2 <= kRankSortMax ? (size_t)2 * n2 * 8 : 0;
  return sel > stage ? sel : stage;
}
__device__ __forceinline__ int large_region_bytes_dev(int n2, int k2) {
  const int sel = k2 * 12;
  const int stage = n2 <= kRankSortMax ? 2 * n2 * 8 : 0;
  return sel > stage ? sel : stage;
}

// Bytes of dynamic LDS the kernel needs.
size_t large_lds_bytes(int n2, int k2, int kr) {
  return (size_t)2 * n2 * 8 + large_region_bytes(n2, k2) + (size_t)(kr + 1) * 4;
}

struct LargeShared {
  uint32_t hist[256];
  uint64_t ts, ms;   // decided high bits of the threshold key and their mask (score part)
  uint32_t tn, mn;   // the same for the ~id part
  int krem;          // keys still to select at and below the current digit
  int mode;          // 0: walk every candidate; 1: walk and copy the prefix matches; 2: read the copy
  int nsurv;         // keys copied
  int count;         // gathered keys
  int wint[kLargeMaxWaves];
  float wsum[kLargeMaxWaves];
  uint64_t wmax[kLargeMaxWaves];
  int pass0;         // first radix pass (the score bytes before it are shared, see step 3)
};

// Walks one thread's chunk of the flat candidate list, one candidate after the other. The
// current row rank's logit (as a double) and id offset stay in registers; the next column key
// and the next row rank's key and end offset are read one step ahead, so LDS latency overlaps
// the work on the current candidate. Every row rank below kr holds at least one candidate,
// so a step moves at most one row rank on.
struct CandWalk {
  const uint64_t* rk;
  const uint64_t* ck;
  const uint32_t* cum;
  int kr, nc;
  int ra, rb, rend;
  double vr;
  uint32_t rid;
  uint64_t cv;     // column key of the current candidate
  uint64_t rnext;  // key of row rank ra + 1
  int rend_next;   // end offset of row rank ra + 1

  __device__ __forceinline__ void set_row(uint64_t r) {
    vr = (double)f32_from_ord((uint32_t)(r >> 32));
    rid = (0xFFFFFFFFu - (uint32_t)r) * (uint32_t)nc;
  }
  __device__ __forceinline__ void prefetch_row() {
    if (ra + 1 < kr) {
      rnext = rk[ra + 1];
      rend_next = (int)cum[ra + 2];
    }
  }
  // Positions the walk at candidate c0 of row rank a_first (c0 < P).
  __device__ __forceinline__ void start(int a_first, int c0) {
    ra = a_first;
    rb = c0 - (int)cum[ra];
    rend = (int)cum[ra + 1];
    set_row(rk[ra]);
    cv = ck[rb];
    prefetch_row();
  }
  // Key of candidate c, then a step to c + 1 (c < P; called for consecutive c).
  __device__ __forceinline__ void next(int c, uint64_t* ks, uint32_t* kn) {
    *ks = ord_f64(vr + (double)f32_from_ord((uint32_t)(cv >> 32)));
    *kn = 0xFFFFFFFFu - (rid + (0xFFFFFFFFu - (uint32_t)cv));
    if (c + 1 >= rend) {
      if (ra + 1 < kr) {
        ++ra;
        rb = 0;
        rend = rend_next;
        set_row(rnext);
        prefetch_row();
      }
    } else {
      ++rb;
    }
    cv = ck[rb];  // in bounds also past the last candidate (rb stays below kc)
  }
};

// Wave-aggregated append: lanes with take set store (ks, kn) at consecutive slots of
// (dst_s, dst_n) reserved with one LDS atomic on *counter. Every lane of the wave calls it.
__device__ __forceinline__ void wave_append(bool take, uint64_t ks, uint32_t kn, int* counter,
                                            uint64_t* dst_s, uint32_t* dst_n, int cap) {
  const uint64_t bal = __ballot(take);
  if (bal == 0ull) return;
  int base = 0;
  if (lane_id() == 0) base = atomicAdd(counter, (int)__popcll(bal));
  base = __builtin_amdgcn_readfirstlane(base);  // lane 0 is active: every lane calls this
  if (take) {
    const int pos = base + (int)__popcll(bal & lanemask_lt());
    if (pos < cap) {
      dst_s[pos] = ks;
      dst_n[pos] = kn;
    }
  }
}

// One radix step, run by all lanes of one wave once the histogram of the current digit is
// complete: the largest digit whose count of keys at or above it reaches krem becomes part of
// the threshold. Lane l reads bins 4l .. 4l + 3. Also advances the survivor-copy mode.
__device__ __forceinline__ void pick_digit(LargeShared& sh, int pass, int mode, int k2) {
  const int l = lane_id();
  const int sh_s = 56 - 8 * pass;
  const int sh_n = 24 - 8 * (pass - 8);
  const int krem = sh.krem;
  const uint32_t h0 = sh.hist[4 * l], h1 = sh.hist[4 * l + 1];
  const uint32_t h2 = sh.hist[4 * l + 2], h3 = sh.hist[4 * l + 3];
  const int mine = (int)(h0 + h1 + h2 + h3);
  // suffix sum over lanes >= l
  int suf = mine;
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    const int y = __shfl_down(suf, m, kWave);
    if (l + m < kWave) suf += y;
  }
  const int above = suf - mine;  // keys in bins of higher lanes
  const uint64_t hit = __ballot(suf >= krem && above < krem);
  const int L = __ffsll((unsigned long long)hit) - 1;
  if (l == L) {
    // within the lane, from bin 4l + 3 down
    int acc = above, dg;
    uint32_t in_bin;
    if (acc + (int)h3 >= krem) {
      dg = 4 * l + 3;
      in_bin = h3;
    } else {
      acc += (int)h3;
      if (acc + (int)h2 >= krem) {
        dg = 4 * l + 2;
        in_bin = h2;
      } else {
        acc += (int)h2;
        if (acc + (int)h1 >= krem) {
          dg = 4 * l + 1;
          in_bin = h1;
        } else {
          acc += (int)h1;
          dg = 4 * l;
          in_bin = h0;
        }
      }
    }
    sh.krem = krem - acc;
    if (pass < 8) {
      sh.ts |= (uint64_t)dg << sh_s;
      sh.ms |= (uint64_t)0xFF << sh_s;
    } else {
      sh.tn |= (uint32_t)dg << sh_n;
      sh.mn |= 0xFFu << sh_n;
    }
    // the copy is taken by the pass after the one whose chosen bin first fits
    sh.mode = mode == 1 ? 2 : ((mode == 0 && (int)in_bin <= k2) ? 1 : mode);
  }
}

// Histogram of the current digit over the survivor copy, threads tid, tid + stride, ...
__device__ __forceinline__ void survivor_hist(LargeShared& sh, const uint64_t* sel_s,
                                              const uint32_t* sel_n, int n, int pass, int tid,
                                              int stride) {
  const uint64_t ts = sh.ts, ms = sh.ms;
  const uint32_t tn = sh.tn, mn = sh.mn;
  const int sh_s = 56 - 8 * pass;
  const int sh_n = 24 - 8 * (pass - 8);
  for (int i = tid; i < n; i += stride) {
    const uint64_t ks = sel_s[i];
    const uint32_t kn = sel_n[i];
    if ((ks & ms) == ts && (kn & mn) == tn) {
      const uint32_t dg = pass < 8 ? (uint32_t)(ks >> sh_s) & 0xFFu : (kn >> sh_n) & 0xFFu;
      atomicAdd(&sh.hist[dg], 1u);
    }
  }
}

// Bitonic merges k = k_lo, 2 k_lo, ..., k_hi (k_hi <= 8) restricted to partner distances below
// 8, on blocks of eight consecutive keys (block b of k2 / 8 held by one thread in registers):
// for each merge, distances min(k / 2, 4), ..., 1; keys are ordered descending by (s, n) where
// (i & k) == 0, ascending elsewhere, as in the LDS levels.
__device__ __forceinline__ void sort_block8(uint64_t* ks, uint32_t* kn, int k2, int k_lo,
                                            int k_hi, int tid, int nthreads) {
  for (int b = tid; b < (k2 >> 3); b += nthreads) {
    uint64_t s[8];
    uint32_t n[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      s[q] = ks[8 * b + q];
      n[q] = kn[8 * b + q];
    }
    for (int k = k_lo; k <= k_hi; k <<= 1) {
#pragma unroll
      for (int j = 4; j >= 1; j >>= 1) {
        if (j >= k) continue;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (q & j) continue;
          const bool up = ((8 * b + q) & k) == 0;
          const bool lt = s[q] < s[q + j] || (s[q] == s[q + j] && n[q] < n[q + j]);
          if (lt == up) {
            const uint64_t ts = s[q];
            s[q] = s[q + j];
            s[q + j] = ts;
            const uint32_t tn = n[q];
            n[q] = n[q + j];
            n[q + j] = tn;
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      ks[8 * b + q] = s[q];
      kn[8 * b + q] = n[q];
    }
  }
}

// Writes the keep largest of the n distinct keys src[0, n) to dst in descending order: the
// rank of a key is the number of larger keys. src is padded with 0 to an even length and
// 16-byte aligned; thread t of NT ranks keys t, t + NT, ...
template <int NT>
__device__ __forceinline__ void rank_half(const uint64_t* src, int n, int keep, int t,
                                          uint64_t* dst) {
  constexpr int kStride = NT;
  constexpr int S = kRankSortMax / kStride;
  uint64_t key[S];
  int rank[S];
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int j = t + kStride * s;
    key[s] = j < n ? src[j] : ~0ull;
    rank[s] = 0;
  }
  const int n_even = (n + 1) & ~1;
#pragma unroll 4
  for (int q = 0; q < n_even; q += 2) {
    const ulonglong2 p = *reinterpret_cast<const ulonglong2*>(src + q);
#pragma unroll
    for (int s = 0; s < S; ++s) rank[s] += (p.x > key[s] ? 1 : 0) + (p.y > key[s] ? 1 : 0);
  }
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int j = t + kStride * s;
    if (j < n && rank[s] < keep) dst[rank[s]] = key[s];
  }
}

template <int NT>
__global__ __launch_bounds__(NT, NT == 256 ? 5 : 4) void select_large_kernel(LargeArgs a) {
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
  uint32_t* cum = (uint32_t*)((unsigned char*)sel_s + large_region_bytes_dev(n2, k2));  // [kr + 1]
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;

  // candidate offsets: cum[a] = sum over a' < a of min(kc, K / (a' + 1)), by a block scan
  {
    const int per = (kr + kLargeThreads - 1) / kLargeThreads;
    const int a0 = tid * per;
    int loc = 0;
    for (int q = a0; q < a0 + per && q < kr; ++q) {
      const int c = K / (q + 1);
      loc += c < kc ? c : kc;
    }
    const int ex = wave_excl_scan_i32(loc);
    if (l == kWave - 1) sh.wint[w] = ex + loc;
    __syncthreads();
    int off = 0;
    for (int ww = 0; ww < w; ++ww) off += sh.wint[ww];
    int run = off + ex;
    for (int q = a0; q < a0 + per && q < kr; ++q) {
      cum[q] = (uint32_t)run;
      const int c = K / (q + 1);
      run += c < kc ? c : kc;
    }
    if (a0 < kr && a0 + per >= kr) cum[kr] = (uint32_t)run;
    __syncthreads();
  }
  const int P = (int)cum[kr];
  const int chunk = (P + kLargeThreads - 1) / kLargeThreads;  // same on every thread
  const int c0 = tid * chunk;
  const int c1 = c0 + chunk < P ? c0 + chunk : P;
  // first row rank of this thread's chunk (binary search in cum)
  int a_first = 0;
  if (c0 < P) {
    int lo = 0, hi = kr - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((int)cum[mid] <= c0) lo = mid; else hi = mid - 1;
    }
    a_first = lo;
  }

  for (int64_t row = blockIdx.x; row < a.rows; row += gridDim.x) {
    const float* hr = a.hs + row * (int64_t)(a.nr + a.nc);
    // 1. the top kr row keys and top kc column keys, descending
    if (n2 <= kRankSortMax) {
      uint64_t* stage = sel_s;  // [2][n2], unsorted, padded with 0 (below every finite logit)
      for (int i = tid; i < 2 * n2; i += kLargeThreads) {
        const int h = i >= n2, j = i - h * n2;
        const int n = h ? a.nc : a.nr;
        stage[i] = j < n ? logit_key(ord_f32(hr[h * a.nr + j]), j) : 0ull;
      }
      __syncthreads();
      rank_half<NT>(stage, a.nr, kr, tid, hk);
      rank_half<NT>(stage + n2, a.nc, kc, tid, hk + n2);
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
    CandWalk walk;
    walk.rk = hk;
    walk.ck = hk + n2;
    walk.cum = cum;
    walk.kr = kr;
    walk.nc = a.nc;
    // 3. radix select of the K-th largest candidate key, eight bits at a time from the top.
    // The leading score bytes that every key at or above the threshold shares are skipped: the
    // largest score is row rank 0 plus column rank 0, and any A x B corner of the sorted grid
    // with A B >= K holds K cells at or above its last cell, so r[A - 1] + c[B - 1] is at most
    // the K-th largest score. All keys between the two share their common leading bytes, and no
    // key lies above the largest, so the search starts below those bytes with krem = K.
    {
      const int amin = (K + kc - 1) / kc;
      uint64_t lo = 0ull;
      for (int A = amin + tid; A <= kr; A += kLargeThreads) {
        const int Bn = (K + A - 1) / A;  // <= kc
        const double v = (double)f32_from_ord((uint32_t)(hk[A - 1] >> 32)) +
                         (double)f32_from_ord((uint32_t)(hk[n2 + Bn - 1] >> 32));
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
      if (tid == 0) {
        for (int ww = 1; ww < kLargeWaves; ++ww) lo = sh.wmax[ww] > lo ? sh.wmax[ww] : lo;
        const uint64_t hi = ord_f64((double)f32_from_ord((uint32_t)(hk[0] >> 32)) +
                                    (double)f32_from_ord((uint32_t)(hk[n2] >> 32)));
        const uint64_t diff = hi ^ lo;
        const int same = diff == 0ull ? 8 : (int)(__clzll((long long)diff) >> 3);
        const uint64_t mask = same == 0 ? 0ull : (same == 8 ? ~0ull : ~0ull << (64 - 8 * same));
        sh.ts = hi & mask;
        sh.ms = mask;
        sh.pass0 = same;
        sh.tn = 0u;
        sh.mn = 0u;
        sh.krem = K;
        sh.mode = 0;
        sh.nsurv = 0;
        sh.count = 0;
      }
      __syncthreads();
    }
    int pass = sh.pass0;
    for (; pass < 12; ++pass) {
      for (int i = tid; i < 256; i += kLargeThreads) sh.hist[i] = 0u;
      __syncthreads();
      const uint64_t ts = sh.ts, ms = sh.ms;
      const uint32_t tn = sh.tn, mn = sh.mn;
      const int mode = sh.mode;
      const int nsurv = sh.nsurv < k2 ? sh.nsurv : k2;
      if (mode == 2 && nsurv <= kWaveFinish) break;  // the same on every thread
      const int sh_s = 56 - 8 * pass;            // digit position in the score word (pass < 8)
      const int sh_n = 24 - 8 * (pass - 8);      // digit position in the id word (pass >= 8)
      if (mode == 2) {
        survivor_hist(sh, sel_s, sel_n, nsurv, pass, tid, kLargeThreads);
      } else {
        // runs of equal digits along the chunk are counted before one LDS atomic, so bins that
        // nearly every candidate hits are not serialised over all of them
        uint32_t run_dg = 0u, run_n = 0u;
        if (c0 < P) walk.start(a_first, c0);
        for (int it = 0; it < chunk; ++it) {
          const int c = c0 + it;
          const bool live = c < c1;
          uint64_t ks = 0ull;
          uint32_t kn = 0u;
          if (live) walk.next(c, &ks, &kn);
          const bool match = live && (ks & ms) == ts && (kn & mn) == tn;
          if (match) {
            const uint32_t dg = pass < 8 ? (uint32_t)(ks >> sh_s) & 0xFFu : (kn >> sh_n) & 0xFFu;
            if (run_n != 0u && dg != run_dg) {
              atomicAdd(&sh.hist[run_dg], run_n);
              run_n = 0u;
            }
            run_dg = dg;
            ++run_n;
          }
          if (mode == 1) wave_append(match, ks, kn, &sh.nsurv, sel_s, sel_n, k2);
        }
        if (run_n != 0u) atomicAdd(&sh.hist[run_dg], run_n);
      }
      __syncthreads();
      if (w == 0) pick_digit(sh, pass, mode, k2);
      __syncthreads();
    }
    if (pass < 12) {
      // a short survivor copy: wave 0 alone takes the remaining digits, with no workgroup
      // barriers between them
      if (w == 0) {
        const int nsurv = sh.nsurv < k2 ? sh.nsurv : k2;
        for (; pass < 12; ++pass) {
          for (int i = l; i < 256; i += kWave) sh.hist[i] = 0u;
          wave_lds_sync();
          survivor_hist(sh, sel_s, sel_n, nsurv, pass, l, kWave);
          wave_lds_sync();
          pick_digit(sh, pass, 2, k2);
          wave_lds_sync();
        }
      }
      __syncthreads();
    }
    // 4. the threshold key is exact now; gather the K keys at or above it
    {
      const uint64_t ts = sh.ts;
      const uint32_t tn = sh.tn;
      if (c0 < P) walk.start(a_first, c0);
      for (int it = 0; it < chunk; ++it) {
        const int c = c0 + it;
        const bool live = c < c1;
        uint64_t ks = 0ull;
        uint32_t kn = 0u;
        if (live) walk.next(c, &ks, &kn);
        const bool take = live && (ks > ts || (ks == ts && kn >= tn));
        wave_append(take, ks, kn, &sh.count, sel_s, sel_n, k2);
      }
      for (int i = K + tid; i < k2; i += kLargeThreads) {
        sel_s[i] = 0ull;
        sel_n[i] = 0u;
      }
    }
    __syncthreads();
    // bitonic sort of the K selected keys, descending by (score, ~id). With eight waves (2048 keys
    // or more) the levels with partner distance 8 or more run over LDS, one compare-exchange
    // per pair, and the last three levels of each merge (distances 4, 2, 1), and the whole of
    // the first three merges, run on eight consecutive keys held in one thread's registers: one
    // LDS pass instead of three. With four waves every level runs over LDS (registers are kept
    // for occupancy there).
    constexpr int kRegFrom = NT == 512 ? 4 : 1;  // first merge whose low levels use registers
    if constexpr (NT == 512) {
      sort_block8(sel_s, sel_n, k2, 2, 8, tid, kLargeThreads);
      __syncthreads();
    }
    for (int lk = kRegFrom; (1 << lk) <= k2; ++lk) {
      const int k = 1 << lk;
      for (int lj = lk - 1; lj >= (NT == 512 ? 3 : 0); --lj) {
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
      if constexpr (NT == 512) {
        sort_block8(sel_s, sel_n, k2, k, k, tid, kLargeThreads);
        __syncthreads();
      }
    }
    // 5. gates: e_k = exp(S_k - S_0), summed per thread over a contiguous range, then across
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
    // eight waves per row once the final sort has 2048 keys or more; four below, where more
    // rows share a compute unit
    if (k2 >= 2048)
      hipLaunchKernelGGL(select_large_kernel<512>, grid, dim3(512), lds, st, a);
    else
      hipLaunchKernelGGL(select_large_kernel<256>, grid, dim3(256), lds, st, a);
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
