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
// Per-half top-K: each lane holds ceil(n / 64) logits. The K-th largest of the 64 lane
// maxima, theta, is at most the K-th largest logit (K distinct lanes hold a value >= theta),
// so the logits >= theta contain the answer. Usually a few more than K of them exist; they are
// compacted into one per lane and bitonic-sorted. When more than 64 qualify (heavy ties), the
// row falls back to sorting them in batches of 64 and merging.
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

// 96-bit key of a grid cell: score (order map of the double) then lower id first.
struct CellKey {
  uint64_t s;
  uint32_t nn;  // ~id, so larger is better
};

__device__ __forceinline__ bool cell_gt(const CellKey& a, const CellKey& b) {
  return a.s > b.s || (a.s == b.s && a.nn > b.nn);
}

__device__ __forceinline__ CellKey shfl_xor_cell(const CellKey& k, int m) {
  CellKey o;
  o.s = shfl_xor_u64(k.s, m);
  o.nn = (uint32_t)__shfl_xor((int)k.nn, m, kWave);
  return o;
}

// Bitonic sort of one key per lane into descending lane order.
__device__ __forceinline__ uint32_t sort_desc_u32(uint32_t v) {
  const int l = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      uint32_t o = (uint32_t)__shfl_xor((int)v, j, kWave);
      bool keep_max = (((l & j) == 0) == ((l & k) == 0));
      v = keep_max ? (v > o ? v : o) : (v < o ? v : o);
    }
  }
  return v;
}

__device__ __forceinline__ uint64_t sort_desc_u64(uint64_t v) {
  const int l = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      uint64_t o = shfl_xor_u64(v, j);
      bool keep_max = (((l & j) == 0) == ((l & k) == 0));
      v = keep_max ? (v > o ? v : o) : (v < o ? v : o);
    }
  }
  return v;
}

// Top 64 of two descending lane-sorted lists, descending.
__device__ __forceinline__ uint64_t merge_desc_u64(uint64_t a, uint64_t b) {
  const int l = lane_id();
  uint64_t rb = shfl_u64(b, (kWave - 1) - l);
  uint64_t v = a > rb ? a : rb;
#pragma unroll
  for (int j = kWave >> 1; j > 0; j >>= 1) {
    uint64_t o = shfl_xor_u64(v, j);
    v = ((l & j) == 0) ? (v > o ? v : o) : (v < o ? v : o);
  }
  return v;
}

__device__ __forceinline__ CellKey sort_desc_cell(CellKey v) {
  const int l = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      CellKey o = shfl_xor_cell(v, j);
      bool keep_max = (((l & j) == 0) == ((l & k) == 0));
      bool gt = cell_gt(v, o);
      v = (keep_max == gt) ? v : o;
    }
  }
  return v;
}

__device__ __forceinline__ CellKey merge_desc_cell(CellKey a, CellKey b) {
  const int l = lane_id();
  CellKey rb;
  rb.s = shfl_u64(b.s, (kWave - 1) - l);
  rb.nn = (uint32_t)__shfl((int)b.nn, (kWave - 1) - l, kWave);
  CellKey v = cell_gt(a, rb) ? a : rb;
#pragma unroll
  for (int j = kWave >> 1; j > 0; j >>= 1) {
    CellKey o = shfl_xor_cell(v, j);
    bool gt = cell_gt(v, o);
    v = (((l & j) == 0) == gt) ? v : o;
  }
  return v;
}

// Key of logit j: value order in the high word, ~j in the low word (ties to lower j).
__device__ __forceinline__ uint64_t logit_key(uint32_t ord, int j) {
  return ((uint64_t)ord << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)j);
}

// Top kh of the n logits at p; lane l < kh receives the l-th best as a logit key.
template <int R>
__device__ uint64_t half_topk(const float* __restrict__ p, int n, int kh, uint64_t* wbuf) {
  const int l = lane_id();
  uint32_t o[R];
  uint32_t mx = 0u;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int j = l + kWave * r;
    o[r] = (j < n) ? ord_f32(p[j]) : 0u;  // 0 sits below every finite value
    mx = o[r] > mx ? o[r] : mx;
  }
  const uint32_t theta = (uint32_t)__shfl((int)sort_desc_u32(mx), kh - 1, kWave);
  int cnt = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) cnt += (o[r] >= theta) ? 1 : 0;
  const int total = wave_sum_i32(cnt);
  if (total <= kWave) {
    int pos = wave_excl_scan_i32(cnt);
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (o[r] >= theta) wbuf[pos++] = logit_key(o[r], l + kWave * r);
    wave_lds_sync();
    uint64_t key = (l < total) ? wbuf[l] : 0ull;
    wave_lds_sync();
    return sort_desc_u64(key);
  }
  uint64_t best = 0ull;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    uint64_t key = (o[r] >= theta) ? logit_key(o[r], l + kWave * r) : 0ull;
    best = merge_desc_u64(best, sort_desc_u64(key));
  }
  return best;
}

template <int R>
__global__ __launch_bounds__(256) void select_kernel(SelectArgs a) {
  __shared__ uint16_t cand[kMaxCand];  // (a << 8) | b
  __shared__ int n_cand;
  __shared__ uint64_t wbuf_all[4][kWave];
  const int K = a.K;
  const int kr = K < a.nr ? K : a.nr;
  const int kc = K < a.nc ? K : a.nc;
  if (threadIdx.x == 0) {
    int c = 0;
    for (int ra = 0; ra < kr; ++ra)
      for (int rb = 0; rb < kc && (ra + 1) * (rb + 1) <= K; ++rb) cand[c++] = (uint16_t)((ra << 8) | rb);
    n_cand = c;
  }
  __syncthreads();
  const int P = n_cand;
  const int l = lane_id();
  const int w = threadIdx.x >> 6;
  uint64_t* wbuf = wbuf_all[w];
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t row = (int64_t)blockIdx.x * 4 + w; row < a.rows; row += stride) {
    const float* hr = a.hs + row * (int64_t)(a.nr + a.nc);
    const uint64_t rk = half_topk<R>(hr, a.nr, kr, wbuf);
    const uint64_t ck = half_topk<R>(hr + a.nr, a.nc, kc, wbuf);
    // Cartesian candidates, 64 per batch.
    CellKey best;
    best.s = 0ull;
    best.nn = 0u;
    for (int base = 0; base < P; base += kWave) {
      int c = base + l;
      int ca = 0, cb = 0;
      if (c < P) {
        ca = cand[c] >> 8;
        cb = cand[c] & 0xFF;
      }
      uint64_t kr_c = shfl_u64(rk, ca);
      uint64_t kc_c = shfl_u64(ck, cb);
      CellKey key;
      key.s = 0ull;
      key.nn = 0u;
      if (c < P) {
        float vr = f32_from_ord((uint32_t)(kr_c >> 32));
        float vc = f32_from_ord((uint32_t)(kc_c >> 32));
        uint32_t i = 0xFFFFFFFFu - (uint32_t)kr_c;
        uint32_t j = 0xFFFFFFFFu - (uint32_t)kc_c;
        key.s = ord_f64((double)vr + (double)vc);
        key.nn = 0xFFFFFFFFu - (i * (uint32_t)a.nc + j);
      }
      key = sort_desc_cell(key);
      best = (base == 0) ? key : merge_desc_cell(best, key);
    }
    // Gates: softmax over the K selected scores, best first.
    const double s = f64_from_ord(best.s);
    const double s0 = __shfl(s, 0, kWave);
    float e = (l < K) ? expf((float)(s - s0)) : 0.0f;
    const float z = wave_sum_f32(e);
    if (l < K) {
      a.idx[row * K + l] = (int32_t)(0xFFFFFFFFu - best.nn);
      a.gates[row * K + l] = e / z;
    }
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
  if (blocks > 4096) blocks = 4096;
  dim3 grid((unsigned)blocks), block(256);
  if (nmax <= 64)
    hipLaunchKernelGGL(select_kernel<1>, grid, block, 0, st, a);
  else if (nmax <= 128)
    hipLaunchKernelGGL(select_kernel<2>, grid, block, 0, st, a);
  else if (nmax <= 256)
    hipLaunchKernelGGL(select_kernel<4>, grid, block, 0, st, a);
  else if (nmax <= 512)
    hipLaunchKernelGGL(select_kernel<8>, grid, block, 0, st, a);
  else if (nmax <= 1024)
    hipLaunchKernelGGL(select_kernel<16>, grid, block, 0, st, a);
  else if (nmax <= 2048)
    hipLaunchKernelGGL(select_kernel<32>, grid, block, 0, st, a);
  else
    hipLaunchKernelGGL(select_kernel<64>, grid, block, 0, st, a);
  return hipGetLastError();
}

}  // namespace omnimoe
