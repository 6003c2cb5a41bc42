// Expert-Centric Scheduling (Sec. 2.3, Eq. 12-13) as a stable least-significant-digit radix
// sort of the task ids p = 0 .. M-1 by expert id idx[p], followed by segment extraction.
//
// Each pass (digit of up to 10 bits) is three steps:
//   upsweep   per-tile digit histogram (tile = 4096 tasks), stored digit-major;
//   scan      exclusive scan of the histogram: the first output slot of (digit, tile);
//   downsweep each wave ranks its tasks stably (ballot-matched peers in lane order plus a
//             per-wave running count); the tile is put in digit order in LDS and each digit's
//             tasks leave as one run, at scan + wave offset + rank.
// Stability of every pass makes the final order (expert, task id), which is unique.
// Segment extraction marks positions whose expert differs from the previous one and
// compacts them with another scan into active / active_offsets / n_active.
// Groups of B > 1 active experts (Eq. 13): each task gets the key q = rank(expert) / B, rank
// being the expert's place in the active list, and a second stable radix sort of the task ids
// by q gives the order (group, task id). Groups are unions of consecutive experts, so
// active_offsets[q B] still marks where group q starts.
// Up to 8192 tasks (decode) take single-launch paths instead: one 16-wave workgroup sorts up to
// 4096 tasks in LDS; from 4097 to 8192 the tasks are split over workgroups by ranges of expert
// ids and a second launch places the segment heads (both further down).
// Everything is integer arithmetic; the LDS atomics only count.
#include <algorithm>
#include <climits>

#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;   // tasks per tile, 1024 per wave
constexpr int kMaxDigitBits = 10;
constexpr int kMaxRadix = 1 << kMaxDigitBits;

// ------------------------------------------------------------------ generic scan
// Exclusive scan over a virtual int array given by a functor, in chunks of kTile.

struct ArrayVal {
  const int32_t* a;
  int64_t n;
  __device__ int operator()(int64_t i) const { return i < n ? a[i] : 0; }
};

struct HeadFlag {  // 1 where a new expert segment starts in the sorted keys
  const int32_t* k;
  int64_t n;
  __device__ int operator()(int64_t i) const {
    if (i >= n) return 0;
    return (i == 0 || k[i] != k[i - 1]) ? 1 : 0;
  }
};

// Block-wide exclusive scan of per-thread values; returns the block total in *total.
__device__ int block_excl_scan(int v, int* total) {
  __shared__ int wsum[kThreads / kWave];
  const int l = lane_id(), w = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    int y = __shfl_up(incl, m, kWave);
    if (l >= m) incl += y;
  }
  if (l == kWave - 1) wsum[w] = incl;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) {
    int s = wsum[i];
    if (i < w) off += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return off + incl - v;
}

// The values of a thread's kItems consecutive items, one call of f each; functors over
// arrays that can do better (vector loads) overload this.
template <class F>
__device__ __forceinline__ void eval_items(const F& f, int64_t base, int (&v)[kItems]) {
#pragma unroll
  for (int j = 0; j < kItems; ++j) v[j] = f(base + j);
}

// HeadFlag over a full interior run: keys base - 1 .. base + kItems - 1 with 16-byte loads.
__device__ __forceinline__ void eval_items(const HeadFlag& f, int64_t base, int (&v)[kItems]) {
  if (base <= 0 || base + kItems > f.n) {
#pragma unroll
    for (int j = 0; j < kItems; ++j) v[j] = f(base + j);
    return;
  }
  int32_t k[kItems + 1];
  k[0] = f.k[base - 1];
#pragma unroll
  for (int q = 0; q < kItems / 4; ++q) {
    const int4 kk = *(const int4*)(f.k + base + 4 * q);
    k[1 + 4 * q] = kk.x; k[2 + 4 * q] = kk.y; k[3 + 4 * q] = kk.z; k[4 + 4 * q] = kk.w;
  }
#pragma unroll
  for (int j = 0; j < kItems; ++j) v[j] = k[j + 1] != k[j] ? 1 : 0;
}

template <class F>
__global__ __launch_bounds__(kThreads) void scan_reduce_kernel(F f, int64_t n, int32_t* partial) {
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
  int v[kItems];
  eval_items(f, base, v);
  int s = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) s += v[j];
  int total;
  block_excl_scan(s, &total);
  if (threadIdx.x == 0) partial[blockIdx.x] = total;
}

// Writes the exclusive scan of f to out (ArrayVal) ...
struct EmitScan {
  int32_t* out;
  int64_t n;
  __device__ void operator()(int64_t i, int val, int pos) const {
    (void)val;
    if (i < n) out[i] = pos;
  }
  __device__ void finish(int total) const { (void)total; }
};

// ... or compacts segment heads into active / active_offsets (HeadFlag) and closes the list:
// n_active and the end offset M. `cap` bounds the output arrays, which only matters if some id
// lies outside [0, N).
struct EmitSegments {
  const int32_t* keys;
  int32_t* active;
  int32_t* offsets;
  int32_t* n_active;
  int32_t cap;
  int32_t m;
  __device__ void operator()(int64_t i, int val, int pos) const {
    if (val && pos < cap) {
      active[pos] = keys[i];
      offsets[pos] = (int32_t)i;
    }
  }
  __device__ void finish(int total) const {
    const int n = total < cap ? total : cap;
    *n_active = n;
    offsets[n] = m;
  }
};

// Second step of the scan: each block first adds up the chunk totals of the blocks before it
// (at most a few hundred values), so no separate pass over the totals is needed. The last
// block hands the grand total to emit.finish.
// This thread's share of partial[0 .. nb): four loads in flight per round (clamped addresses,
// masked values) rather than one load and wait per value.
__device__ __forceinline__ int partial_prefix(const int32_t* partial, int nb) {
  int pre = 0;
  for (int i0 = 0; i0 < nb; i0 += 4 * kThreads) {
    int a[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kThreads + (int)threadIdx.x;
      a[u] = partial[i < nb ? i : nb - 1];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) pre += i0 + u * kThreads + (int)threadIdx.x < nb ? a[u] : 0;
  }
  return pre;
}

template <class F, class E>
__global__ __launch_bounds__(kThreads) void scan_down_kernel(F f, E emit, const int32_t* partial) {
  int before;
  block_excl_scan(partial_prefix(partial, (int)blockIdx.x), &before);
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
  int v[kItems];
  eval_items(f, base, v);
  int s = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) s += v[j];
  int total;
  int pos = block_excl_scan(s, &total) + before;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    emit(base + j, v[j], pos);
    pos += v[j];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) emit.finish(before + total);
}

template <class F, class E>
hipError_t device_scan(F f, E emit, int64_t n, int32_t* partial, hipStream_t st) {
  const int nb = (int)((n + kTile - 1) / kTile);
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL(scan_reduce_kernel<F>, dim3(nb), dim3(kThreads), 0, st, f, n, partial);
  hipLaunchKernelGGL((scan_down_kernel<F, E>), dim3(nb), dim3(kThreads), 0, st, f, emit,
                     (const int32_t*)partial);
  return hipGetLastError();
}

// ------------------------------------------------------------------ radix pass

struct RadixPass {
  const int32_t* keys_in;
  const int32_t* vals_in;  // NULL: values are the positions (task ids)
  int32_t* keys_out;
  int32_t* vals_out;
  int32_t* hist;           // [radix][num_tiles]
  int64_t n;
  int shift, bits, num_tiles;
};

__global__ __launch_bounds__(kThreads) void radix_upsweep_kernel(RadixPass p) {
  __shared__ int cnt[kMaxRadix];
  const int radix = 1 << p.bits;
  for (int d = threadIdx.x; d < radix; d += kThreads) cnt[d] = 0;
  __syncthreads();
  const int64_t tile = xcd_contiguous(blockIdx.x, p.num_tiles);
  const int64_t base = tile * kTile;
  const uint32_t mask = (uint32_t)radix - 1u;
#pragma unroll 4
  for (int j = 0; j < kItems; ++j) {
    int64_t i = base + threadIdx.x + (int64_t)kThreads * j;
    if (i < p.n) atomicAdd(&cnt[((uint32_t)p.keys_in[i] >> p.shift) & mask], 1);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < radix; d += kThreads)
    p.hist[(int64_t)d * p.num_tiles + tile] = cnt[d];
}

__global__ __launch_bounds__(kThreads) void radix_downsweep_kernel(RadixPass p) {
  static_assert(kMaxRadix <= 4 * kThreads, "each thread scans four digits");
  __shared__ int wcnt[kThreads / kWave][kMaxRadix];
  __shared__ int gofs[kMaxRadix];  // first output slot of each digit, then minus its local start
  __shared__ int wsum[kThreads / kWave];
  __shared__ int skey[kTile];
  __shared__ int sval[kTile];
  const int radix = 1 << p.bits;
  const uint32_t mask = (uint32_t)radix - 1u;
  // Tiles in XCD-contiguous order: a digit's runs from neighbouring tiles are adjacent in the
  // output, and written from one L2 they merge into whole lines.
  const int64_t tile = xcd_contiguous(blockIdx.x, p.num_tiles);
  for (int d = threadIdx.x; d < radix; d += kThreads) {
    gofs[d] = p.hist[(int64_t)d * p.num_tiles + tile];
#pragma unroll
    for (int w = 0; w < kThreads / kWave; ++w) wcnt[w][d] = 0;
  }
  __syncthreads();
  const int l = lane_id(), w = threadIdx.x >> 6;
  const int64_t wbase = tile * kTile + (int64_t)w * (kTile / 4);
  const uint64_t lt = lanemask_lt();
  int key[kItems], val[kItems], rank[kItems];
  // All loads first: the LDS fences of the ranking rounds would otherwise hold each round's
  // loads back until the previous round finished.
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int64_t i = wbase + (int64_t)r * kWave + l;
    const bool valid = i < p.n;
    key[r] = valid ? p.keys_in[i] : 0;
    val[r] = valid ? (p.vals_in ? p.vals_in[i] : (int)i) : 0;
  }
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int64_t i = wbase + (int64_t)r * kWave + l;
    const bool valid = i < p.n;
    const uint32_t d = ((uint32_t)key[r] >> p.shift) & mask;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < p.bits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    const int before = __popcll(peers & lt);
    const int count = __popcll(peers);
    int run = valid ? wcnt[w][d] : 0;
    wave_lds_sync();
    if (valid && before == 0) wcnt[w][d] = run + count;
    wave_lds_sync();
    rank[r] = run + before;
  }
  __syncthreads();
  // The tile is first put in digit order in LDS, so that its keys leave as one run per digit
  // (consecutive threads, consecutive addresses) instead of one scattered word per task.
  // With lofs(d) the first local position of digit d, gofs[d] becomes gofs[d] - lofs(d) (a key at
  // local position j goes to gofs[d] + j) and wcnt[ww][d] the local start of wave ww's keys of
  // digit d. Thread t scans digits 4 t .. 4 t + 3. (One array instead of two keeps the LDS at
  // three workgroups per compute unit.)
  {
    int c[4], sum = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int d = 4 * threadIdx.x + k;
      int t = 0;
      if (d < radix) {
#pragma unroll
        for (int ww = 0; ww < kThreads / kWave; ++ww) t += wcnt[ww][d];
      }
      c[k] = t;
      sum += t;
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      const int y = __shfl_up(incl, off, kWave);
      if (l >= off) incl += y;
    }
    if (l == kWave - 1) wsum[w] = incl;
    __syncthreads();
    int base = incl - sum;
    for (int ww = 0; ww < w; ++ww) base += wsum[ww];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int d = 4 * threadIdx.x + k;
      if (d < radix) {
        gofs[d] -= base;
        int run = base;
#pragma unroll
        for (int ww = 0; ww < kThreads / kWave; ++ww) {
          const int cc = wcnt[ww][d];
          wcnt[ww][d] = run;
          run += cc;
        }
      }
      base += c[k];
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kItems; ++r) {
    const int64_t i = wbase + (int64_t)r * kWave + l;
    if (i < p.n) {
      const uint32_t d = ((uint32_t)key[r] >> p.shift) & mask;
      const int lp = wcnt[w][d] + rank[r];
      skey[lp] = key[r];
      sval[lp] = val[r];
    }
  }
  __syncthreads();
  const int64_t t0 = tile * kTile;
  const int tn = (int)(p.n - t0 < kTile ? p.n - t0 : kTile);
  for (int j = threadIdx.x; j < tn; j += kThreads) {
    const int k = skey[j];
    const uint32_t d = ((uint32_t)k >> p.shift) & mask;
    const int64_t pos = (int64_t)gofs[d] + j;
    p.keys_out[pos] = k;
    p.vals_out[pos] = sval[j];
  }
}

// dense[e] = first sorted position of expert e = active_offsets[lower_bound(active, e)].
__global__ __launch_bounds__(kThreads) void dense_offsets_kernel(const int32_t* active,
                                                                 const int32_t* offsets,
                                                                 const int32_t* n_active,
                                                                 int32_t* dense, int64_t n_experts) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e > n_experts) return;
  int lo = 0, hi = *n_active;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if ((int64_t)active[mid] < e) lo = mid + 1; else hi = mid;
  }
  dense[e] = offsets[lo];
}

__global__ __launch_bounds__(kThreads) void fill_i32_kernel(int32_t* dst, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) dst[i] = v;
}

// rank[active[a]] = a for the n_active active experts.
__global__ __launch_bounds__(kThreads) void rank_fill_kernel(const int32_t* active,
                                                            const int32_t* n_active, int32_t* rank,
                                                            int64_t cap, int64_t n_experts) {
  const int64_t a = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (a >= cap || a >= *n_active) return;
  const int32_t e = active[a];
  if (e >= 0 && e < n_experts) rank[e] = (int32_t)a;
}

// ------------------------------------------------------------------ grouped-GEMM plan
// For a schedule with groups of B > 1 experts (tasks in (group, task id) order), a slot is a
// (group, token) pair: the tasks of one token inside one group, contiguous in perm since a
// group's tasks are in task-id (so token) order. Slots are numbered group by group.

__device__ __forceinline__ int32_t clamp_task(int32_t p, int64_t m) {
  return p < 0 ? 0 : (p >= m ? (int32_t)(m - 1) : p);
}

// Division by the runtime constant H K without a divide: q = (umulhi(m, n) + n) >> l with
// l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1 (Granlund and Montgomery), exact for
// 0 <= n < 2^31.
struct DivMagic {
  uint32_t m;
  int l;
};
DivMagic div_magic(uint32_t d) {
  int l = 0;
  while (((uint64_t)1 << l) < d) ++l;
  const uint64_t m = (((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d + 1;
  return DivMagic{(uint32_t)m, l};
}
__device__ __forceinline__ uint32_t div_by(uint32_t n, DivMagic g) {
  return (__umulhi(g.m, n) + n) >> g.l;
}

// Group key of a task of expert e: the expert's rank r in the active list split as
// (r % B) << gb | r / B. The sort reads only the low gb bits, so the expert's place inside its
// group rides along to the sorted order.
__device__ __forceinline__ int32_t group_key_of(int32_t e, const int32_t* rank, int64_t n_experts,
                                                int b, DivMagic bm, int gb) {
  e = e < 0 ? 0 : (e >= n_experts ? (int32_t)(n_experts - 1) : e);
  const uint32_t r = (uint32_t)rank[e];
  const uint32_t q = div_by(r, bm);
  return (int32_t)(((r - q * (uint32_t)b) << gb) | q);
}

constexpr int kKeyItems = 8;  // tasks per thread of the key kernels
unsigned key_blocks(int64_t m) {
  const int64_t per = (int64_t)kThreads * kKeyItems;
  return (unsigned)((m + per - 1) / per);
}

// key[p] = group_key_of(idx[p]) for every task, kKeyItems consecutive tasks per thread: the ids
// with 16-byte loads, then all their rank reads in flight at once (one task per thread would
// leave each wave waiting on one HBM load and one dependent L2 load at a time). idx and key are
// 16-byte aligned.
__global__ __launch_bounds__(kThreads) void group_key_kernel(const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ rank,
                                                            int32_t* __restrict__ key, int64_t m,
                                                            int64_t n_experts, int b, DivMagic bm,
                                                            int gb) {
  const int64_t p0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kKeyItems;
  if (p0 >= m) return;
  if (p0 + kKeyItems <= m) {
    const int4 a = *(const int4*)(idx + p0);
    const int4 c = *(const int4*)(idx + p0 + 4);
    int4 ka, kc;
    ka.x = group_key_of(a.x, rank, n_experts, b, bm, gb);
    ka.y = group_key_of(a.y, rank, n_experts, b, bm, gb);
    ka.z = group_key_of(a.z, rank, n_experts, b, bm, gb);
    ka.w = group_key_of(a.w, rank, n_experts, b, bm, gb);
    kc.x = group_key_of(c.x, rank, n_experts, b, bm, gb);
    kc.y = group_key_of(c.y, rank, n_experts, b, bm, gb);
    kc.z = group_key_of(c.z, rank, n_experts, b, bm, gb);
    kc.w = group_key_of(c.w, rank, n_experts, b, bm, gb);
    *(int4*)(key + p0) = ka;
    *(int4*)(key + p0 + 4) = kc;
    return;
  }
  for (int64_t p = p0; p < m; ++p) key[p] = group_key_of(idx[p], rank, n_experts, b, bm, gb);
}

// The same key for each sorted position of a caller's schedule: key[i] of task perm[i],
// kKeyItems positions per thread (perm with 16-byte loads, the idx and rank reads batched).
__global__ __launch_bounds__(kThreads) void position_key_kernel(const int32_t* __restrict__ perm,
                                                               const int32_t* __restrict__ idx,
                                                               const int32_t* __restrict__ rank,
                                                               int32_t* __restrict__ key,
                                                               int64_t m, int64_t n_experts,
                                                               int b, DivMagic bm, int gb) {
  const int64_t i0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kKeyItems;
  if (i0 >= m) return;
  if (i0 + kKeyItems <= m) {
    const int4 pa = *(const int4*)(perm + i0);
    const int4 pc = *(const int4*)(perm + i0 + 4);
    const int32_t pp[kKeyItems] = {pa.x, pa.y, pa.z, pa.w, pc.x, pc.y, pc.z, pc.w};
    int32_t e[kKeyItems];
#pragma unroll
    for (int j = 0; j < kKeyItems; ++j) e[j] = idx[clamp_task(pp[j], m)];
    int4 ka, kc;
    ka.x = group_key_of(e[0], rank, n_experts, b, bm, gb);
    ka.y = group_key_of(e[1], rank, n_experts, b, bm, gb);
    ka.z = group_key_of(e[2], rank, n_experts, b, bm, gb);
    ka.w = group_key_of(e[3], rank, n_experts, b, bm, gb);
    kc.x = group_key_of(e[4], rank, n_experts, b, bm, gb);
    kc.y = group_key_of(e[5], rank, n_experts, b, bm, gb);
    kc.z = group_key_of(e[6], rank, n_experts, b, bm, gb);
    kc.w = group_key_of(e[7], rank, n_experts, b, bm, gb);
    *(int4*)(key + i0) = ka;
    *(int4*)(key + i0 + 4) = kc;
    return;
  }
  for (int64_t i = i0; i < m; ++i)
    key[i] = group_key_of(idx[clamp_task(perm[i], m)], rank, n_experts, b, bm, gb);
}

// ------------------------------------------------------------------ active experts by bitmap
// For the grouped layer the active list and each expert's rank in it come from a bitmap of the
// experts that have tasks, bit e of word e / 32, instead of a sort by expert. With the bitmap
// and its per-word prefix popcounts in LDS a task's group key needs no global gather:
// rank(e) = prefix[e / 32] + popcount(bits[e / 32] below bit e % 32).

constexpr int kMapWords = 8192;     // largest bitmap kept in LDS with its prefix: 262144 experts
constexpr int kMapThreads = 1024;
constexpr int kMapChunk = kMapThreads * 16;  // tasks per workgroup round, 16 per thread

__device__ __forceinline__ uint32_t clamp_expert(int32_t e, int64_t n_experts) {
  return (uint32_t)(e < 0 ? 0 : (e >= n_experts ? (int32_t)(n_experts - 1) : e));
}

// Sets the bit of the expert of every task (ids clamped into [0, n_experts), as the key kernels
// clamp them). Each workgroup sets the bits of its rounds of tasks in an LDS copy, then ORs the
// copy's nonzero words into bits: one global atomic per word and workgroup instead of a
// scattered store per task. bits holds `words` zeroed words.
__global__ __launch_bounds__(kMapThreads) void mark_experts_kernel(const int32_t* __restrict__ idx,
                                                                  uint32_t* bits, int64_t m,
                                                                  int64_t n_experts, int words) {
  extern __shared__ uint32_t sb[];
  for (int w = threadIdx.x; w < words; w += kMapThreads) sb[w] = 0;
  __syncthreads();
  auto set = [&](int32_t e) {
    const uint32_t c = clamp_expert(e, n_experts);
    atomicOr(&sb[c >> 5], 1u << (c & 31u));
  };
  for (int64_t c0 = (int64_t)blockIdx.x * kMapChunk; c0 < m; c0 += (int64_t)gridDim.x * kMapChunk) {
    if (c0 + kMapChunk <= m) {
      int4 a[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        a[q] = *(const int4*)(idx + c0 + q * (kMapThreads * 4) + threadIdx.x * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        set(a[q].x); set(a[q].y); set(a[q].z); set(a[q].w);
      }
    } else {
      for (int64_t p = c0 + threadIdx.x; p < m; p += kMapThreads) set(idx[p]);
    }
  }
  __syncthreads();
  for (int w = threadIdx.x; w < words; w += kMapThreads)
    if (sb[w]) atomicOr(&bits[w], sb[w]);
}

struct PopWord {  // number of active experts in bitmap word i
  const uint32_t* bits;
  int64_t n;
  __device__ int operator()(int64_t i) const { return i < n ? __popc(bits[i]) : 0; }
};

// Stores each word's exclusive prefix popcount; closes the active list with n_active.
struct EmitPrefix {
  int32_t* prefix;
  int32_t* n_active;
  int64_t n;
  int32_t cap;
  __device__ void operator()(int64_t i, int val, int pos) const {
    (void)val;
    if (i < n) prefix[i] = pos;
  }
  __device__ void finish(int total) const { *n_active = total < cap ? total : cap; }
};

// active[rank(e)] = e for every marked expert e, one thread per expert.
__global__ __launch_bounds__(kThreads) void list_active_kernel(const uint32_t* __restrict__ bits,
                                                              const int32_t* __restrict__ prefix,
                                                              int32_t* __restrict__ active,
                                                              int64_t n_experts, int32_t cap) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= n_experts) return;
  const uint32_t word = bits[e >> 5];
  const uint32_t bit = (uint32_t)e & 31u;
  if (!((word >> bit) & 1u)) return;
  const int32_t r = prefix[e >> 5] + __popc(word & ((1u << bit) - 1u));
  if (r < cap) active[r] = (int32_t)e;
}

// group_key_of for every task with the rank taken from the LDS bitmap and prefix (dynamic LDS of
// 2 * words words); kMapChunk tasks per workgroup round, idx and key 16-byte aligned.
__global__ __launch_bounds__(kMapThreads) void group_key_map_kernel(
    const int32_t* __restrict__ idx, const uint32_t* __restrict__ bits,
    const int32_t* __restrict__ prefix, int32_t* __restrict__ key, int64_t m, int64_t n_experts,
    int words, int b, DivMagic bm, int gb) {
  extern __shared__ uint32_t sm[];
  uint32_t* sb = sm;
  int32_t* sp = (int32_t*)(sm + words);
  for (int w = threadIdx.x; w < words; w += kMapThreads) {
    sb[w] = bits[w];
    sp[w] = prefix[w];
  }
  __syncthreads();
  auto key_of = [&](int32_t e) {
    const uint32_t c = clamp_expert(e, n_experts);
    const uint32_t w = c >> 5;
    const uint32_t r =
        (uint32_t)sp[w] + (uint32_t)__popc(sb[w] & ((1u << (c & 31u)) - 1u));
    const uint32_t q = div_by(r, bm);
    return (int32_t)(((r - q * (uint32_t)b) << gb) | q);
  };
  for (int64_t c0 = (int64_t)blockIdx.x * kMapChunk; c0 < m; c0 += (int64_t)gridDim.x * kMapChunk) {
    if (c0 + kMapChunk <= m) {
      int4 a[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        a[q] = *(const int4*)(idx + c0 + q * (kMapThreads * 4) + threadIdx.x * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int4 k;
        k.x = key_of(a[q].x); k.y = key_of(a[q].y); k.z = key_of(a[q].z); k.w = key_of(a[q].w);
        *(int4*)(key + c0 + q * (kMapThreads * 4) + threadIdx.x * 4) = k;
      }
    } else {
      for (int64_t p = c0 + threadIdx.x; p < m; p += kMapThreads) key[p] = key_of(idx[p]);
    }
  }
}

struct SlotHead {  // 1 where sorted position i starts a new (group, token) slot
  const int32_t* perm;
  const int32_t* key;
  int64_t m;
  uint32_t gmask;
  DivMagic hk;
  __device__ int operator()(int64_t i) const {
    if (i >= m) return 0;
    const int64_t j = i > 0 ? i - 1 : 0;
    const uint32_t p = (uint32_t)clamp_task(perm[i], m);
    const uint32_t p0 = (uint32_t)clamp_task(perm[j], m);
    const uint32_t g = (uint32_t)key[i] ^ (uint32_t)key[j];
    return ((i == 0) | ((g & gmask) != 0u) | (div_by(p, hk) != div_by(p0, hk))) ? 1 : 0;
  }
};

// SlotHead over a full interior run of items: perm and the keys of positions base - 1 ..
// base + kItems - 1 with 16-byte loads (base is a multiple of kItems, the arrays 16-byte
// aligned), the rest as above.
__device__ __forceinline__ void eval_items(const SlotHead& h, int64_t base, int (&v)[kItems]) {
  if (base <= 0 || base + kItems > h.m) {
#pragma unroll
    for (int j = 0; j < kItems; ++j) v[j] = h(base + j);
    return;
  }
  int32_t p[kItems + 1], k[kItems + 1];
  p[0] = h.perm[base - 1];
  k[0] = h.key[base - 1];
#pragma unroll
  for (int q = 0; q < kItems / 4; ++q) {
    const int4 pp = *(const int4*)(h.perm + base + 4 * q);
    const int4 kk = *(const int4*)(h.key + base + 4 * q);
    p[1 + 4 * q] = pp.x; p[2 + 4 * q] = pp.y; p[3 + 4 * q] = pp.z; p[4 + 4 * q] = pp.w;
    k[1 + 4 * q] = kk.x; k[2 + 4 * q] = kk.y; k[3 + 4 * q] = kk.z; k[4 + 4 * q] = kk.w;
  }
  uint32_t t[kItems + 1];
#pragma unroll
  for (int j = 0; j <= kItems; ++j) t[j] = div_by((uint32_t)clamp_task(p[j], h.m), h.hk);
#pragma unroll
  for (int j = 0; j < kItems; ++j)
    v[j] = ((((uint32_t)k[j + 1] ^ (uint32_t)k[j]) & h.gmask) != 0u || t[j + 1] != t[j]) ? 1 : 0;
}

// Outputs of the slot-head scan (slot_heads_down_kernel): every slot's token and first sorted
// position, every group's first slot, the slot count.
struct EmitSlots {
  SlotHead h;
  const int32_t* n_active;
  int64_t groups;
  int b;
  int32_t* slot_token;
  int32_t* slot_off;
  int32_t* grp_slot;
  int32_t* counters;
  __device__ void finish(int total) const {
    slot_off[total] = (int32_t)h.m;
    counters[0] = total;
    const int64_t ng = ((int64_t)*n_active + b - 1) / b;
    grp_slot[ng < groups ? ng : groups] = total;
  }
};

// The slot-head scan's second step with the compaction staged in LDS: each thread keeps the
// token and group key of its items from the flag evaluation, puts its heads' (token, position)
// pairs at their rank inside the tile, and the workgroup writes both lists out as contiguous
// runs (emitting from the items would re-read perm and key for every head and store one
// scattered word per head). Group heads, a few per tile, are written directly.
__global__ __launch_bounds__(kThreads) void slot_heads_down_kernel(EmitSlots e,
                                                                  const int32_t* partial) {
  __shared__ int32_t s_tok[kTile];
  __shared__ int32_t s_off[kTile];
  const SlotHead& h = e.h;
  int before;
  block_excl_scan(partial_prefix(partial, (int)blockIdx.x), &before);
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
  // perm and key at positions base - 1 .. base + kItems - 1 (clamped into [0, m) at the ends)
  int32_t p[kItems + 1], k[kItems + 1];
  if (base > 0 && base + kItems <= h.m) {
    p[0] = h.perm[base - 1];
    k[0] = h.key[base - 1];
#pragma unroll
    for (int q = 0; q < kItems / 4; ++q) {
      const int4 pp = *(const int4*)(h.perm + base + 4 * q);
      const int4 kk = *(const int4*)(h.key + base + 4 * q);
      p[1 + 4 * q] = pp.x; p[2 + 4 * q] = pp.y; p[3 + 4 * q] = pp.z; p[4 + 4 * q] = pp.w;
      k[1 + 4 * q] = kk.x; k[2 + 4 * q] = kk.y; k[3 + 4 * q] = kk.z; k[4 + 4 * q] = kk.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j <= kItems; ++j) {
      int64_t i = base - 1 + j;
      i = i < 0 ? 0 : (i >= h.m ? h.m - 1 : i);
      p[j] = h.perm[i];
      k[j] = h.key[i];
    }
  }
  uint32_t t[kItems + 1];
#pragma unroll
  for (int j = 0; j <= kItems; ++j) t[j] = div_by((uint32_t)clamp_task(p[j], h.m), h.hk);
  int v[kItems], cnt = 0;
  uint32_t gnew = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + j;
    const bool gs = i == 0 || ((((uint32_t)k[j + 1] ^ (uint32_t)k[j]) & h.gmask) != 0u);
    v[j] = (i < h.m && (gs || t[j + 1] != t[j])) ? 1 : 0;
    gnew |= (i < h.m && gs) ? 1u << j : 0u;
    cnt += v[j];
  }
  int total;
  int lp = block_excl_scan(cnt, &total);
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    if (v[j]) {
      s_tok[lp] = (int32_t)t[j + 1];
      s_off[lp] = (int32_t)(base + j);
      const uint32_t g = (uint32_t)k[j + 1] & h.gmask;
      if (((gnew >> j) & 1u) && g < (uint64_t)e.groups) e.grp_slot[g] = before + lp;
    }
    lp += v[j];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < total; i += kThreads) {
    e.slot_token[before + i] = s_tok[i];
    e.slot_off[before + i] = s_off[i];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) e.finish(before + total);
}

struct GroupTiles {  // work tiles of group q: ceil(slots / 256) * ceil(experts / te)
  const int32_t* grp_slot;
  const int32_t* n_active;
  int64_t groups;
  int b, te;
  __device__ int operator()(int64_t q) const {
    const int na = *n_active;
    const int64_t ng = ((int64_t)na + b - 1) / b;
    if (q >= ng || q >= groups) return 0;
    const int tq = grp_slot[q + 1] - grp_slot[q];
    const int64_t bq64 = (int64_t)na - q * b;
    const int bq = bq64 < b ? (int)bq64 : b;
    return ((tq + kGroupSlots - 1) / kGroupSlots) * ((bq + te - 1) / te);
  }
};

struct EmitTiles {
  int32_t* grp_tile;
  int64_t n;
  int32_t* counters;
  __device__ void operator()(int64_t i, int val, int pos) const {
    (void)val;
    if (i < n) grp_tile[i] = pos;
  }
  __device__ void finish(int total) const { counters[1] = total; }
};

size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

int digit_bits_total(int64_t n_experts) {
  int b = 0;
  while ((int64_t)1 << b < n_experts) ++b;
  return b;
}

}  // namespace

// ---------------------------------------------------------------- small task counts
// One workgroup of 16 waves sorts up to 8192 tasks and extracts the segments in a single
// launch (decode shapes). When the keys are spread out (no bucket of the top ten key bits holds
// more than 128 tasks, the usual case), the tasks are counted into those 1024 buckets, placed
// into their bucket's range in any order, and each task's final place is its bucket's start
// plus the number of (expert, task) keys in the bucket below its own: no radix passes. Otherwise
// the multi-kernel path's algorithm runs in LDS: per pass, wave w ranks its contiguous slice of
// tasks stably with ballot-matched peers and per-wave digit counters, the (digit, wave) counts
// are scanned digit-major, and tasks scatter. Either way the segment heads are then counted from
// the sorted keys in LDS and compacted with a block scan.

constexpr int kSmallWaves = 16;
constexpr int kSmallThreads = kSmallWaves * kWave;
constexpr int kSmallRounds = 8;
constexpr int kSmallMax = kSmallThreads * kSmallRounds;  // 8192

struct SmallSched {
  const int32_t* idx;
  int32_t* sorted;  // expert id of each sorted position
  int32_t* perm;
  int32_t* active;
  int32_t* offsets;
  int32_t* n_active;
  int M;
  int cap;
  int passes, per, total_bits;
  // after schedule_ranges_kernel (G > 0): its staged heads, placed here unless a range overflowed
  const int32_t* stage_act;
  const int32_t* stage_off;
  const int32_t* range_base;
  const int32_t* range_heads;
  int G;
};

// Segment heads of the sorted keys in LDS (expert of each sorted position): each thread owns up
// to 8 consecutive positions; the heads are counted, scanned and written to active / offsets.
__device__ void small_heads(const SmallSched& a, const int* skey, int* wsum) {
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  const int per_t = (a.M + kSmallThreads - 1) / kSmallThreads;
  const int b0 = tid * per_t;
  int heads = 0;
  if (per_t == 8 && b0 + 8 <= a.M) {
    // eight consecutive keys with two 16-byte reads (b0 is a multiple of 8)
    const int4 k0 = *(const int4*)(skey + b0);
    const int4 k1 = *(const int4*)(skey + b0 + 4);
    const int pv = b0 > 0 ? skey[b0 - 1] : ~k0.x;
    heads = (k0.x != pv) + (k0.y != k0.x) + (k0.z != k0.y) + (k0.w != k0.z) + (k1.x != k0.w) +
            (k1.y != k1.x) + (k1.z != k1.y) + (k1.w != k1.z);
  } else {
    for (int i = b0; i < b0 + per_t && i < a.M; ++i) heads += (i == 0 || skey[i] != skey[i - 1]);
  }
  const int ex = wave_excl_scan_i32(heads);
  if (l == kWave - 1) wsum[w] = ex + heads;
  __syncthreads();
  int off = 0, tot = 0;
  for (int ww = 0; ww < kSmallWaves; ++ww) {
    const int v = wsum[ww];
    if (ww < w) off += v;
    tot += v;
  }
  int pos = off + ex;
  for (int i = b0; i < b0 + per_t && i < a.M; ++i) {
    if (i == 0 || skey[i] != skey[i - 1]) {
      if (pos < a.cap) {
        a.active[pos] = skey[i];
        a.offsets[pos] = i;
      }
      ++pos;
    }
  }
  if (tid == 0) {
    const int n = tot < a.cap ? tot : a.cap;
    *a.n_active = n;
    a.offsets[n] = a.M;
  }
}

// Outputs of the bucket path from the sorted 64-bit keys in LDS: thread t writes positions
// 8 t .. 8 t + 7 of perm and of the sorted experts with 16-byte stores, keeps the experts in
// LDS for the segment heads, then compacts the heads.
__device__ void small_out_sorted(const SmallSched& a, const uint64_t* keys, int* sorted_lds,
                                 int* wsum) {
  const int tid = threadIdx.x;
  const int b0 = tid * 8;
  if (b0 + 8 <= a.M) {
    int32_t e[8], t[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint64_t k = keys[b0 + q];
      e[q] = (int32_t)(k >> 32);
      t[q] = (int32_t)(uint32_t)k;
    }
    *(int4*)(a.perm + b0) = make_int4(t[0], t[1], t[2], t[3]);
    *(int4*)(a.perm + b0 + 4) = make_int4(t[4], t[5], t[6], t[7]);
    *(int4*)(a.sorted + b0) = make_int4(e[0], e[1], e[2], e[3]);
    *(int4*)(a.sorted + b0 + 4) = make_int4(e[4], e[5], e[6], e[7]);
    *(int4*)(sorted_lds + b0) = make_int4(e[0], e[1], e[2], e[3]);
    *(int4*)(sorted_lds + b0 + 4) = make_int4(e[4], e[5], e[6], e[7]);
  } else {
    for (int i = b0; i < b0 + 8 && i < a.M; ++i) {
      const uint64_t k = keys[i];
      a.perm[i] = (int32_t)(uint32_t)k;
      a.sorted[i] = (int32_t)(k >> 32);
      sorted_lds[i] = (int32_t)(k >> 32);
    }
  }
  __syncthreads();
  small_heads(a, sorted_lds, wsum);
}

// ---------------------------------------------------------------- range-partitioned small sort
// Up to 8192 tasks over many compute units (decode with tens of tokens): workgroup r owns the
// experts [r N / G, (r + 1) N / G). It reads every task id, counts the tasks of lower ranges
// (its first sorted position) and gathers its own (expert, task) keys into LDS; each key's
// place is the number of smaller keys (keys are distinct). It writes its stretch of perm and
// of the sorted experts, and stages its segment heads. schedule_small_kernel then places the
// staged heads (an exclusive scan over the G head counts) with one workgroup. A range that
// holds more than kRangeCap tasks (heavy skew, few experts) reports -1, and
// schedule_small_kernel then sorts everything itself.
constexpr int kRangeThreads = 1024;
constexpr int kRangeCap = 1024;
constexpr int kRangeTasks = 256;  // nominal tasks per range under uniform routing
constexpr int kRangeMinTasks = 4096;  // up to this many tasks: schedule_small_kernel alone
constexpr int kRangeLoads = kSmallMax / kRangeThreads;  // task ids per thread
static_assert(kSmallMax / kRangeTasks <= kWave, "range head counts scanned by one wave");

struct RangeSched {
  const int32_t* idx;
  int32_t* sorted;       // [M] expert of each sorted position
  int32_t* perm;         // [M]
  int32_t* stage_act;    // [M] heads of range r from range_base[r] on: expert
  int32_t* stage_off;    // [M] ... and its first sorted position
  int32_t* range_base;   // [G] tasks in lower ranges
  int32_t* range_heads;  // [G] heads in the range, -1 when it held more than kRangeCap tasks
  int64_t N;
  int M;
  int G;
};

// Exclusive scan of one int per thread over a workgroup of kRangeThreads; *total gets the sum.
__device__ __forceinline__ int range_block_scan(int v, int* wsum, int* total) {
  const int l = lane_id(), w = threadIdx.x >> 6;
  const int ex = wave_excl_scan_i32(v);
  if (l == kWave - 1) wsum[w] = ex + v;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int ww = 0; ww < kRangeThreads / kWave; ++ww) {
    off += ww < w ? wsum[ww] : 0;
    tot += wsum[ww];
  }
  __syncthreads();
  *total = tot;
  return off + ex;
}

__global__ __launch_bounds__(kRangeThreads) void schedule_ranges_kernel(RangeSched a) {
  // gathered keys in any order (padded with ~0 to a multiple of eight), then in order
  __shared__ __attribute__((aligned(16))) uint64_t keys[kRangeCap + 8];
  __shared__ uint64_t sorted[kRangeCap];
  __shared__ int rk[kRangeCap];
  __shared__ int wsum[kRangeThreads / kWave];
  const int tid = threadIdx.x, l = lane_id();
  const int r = blockIdx.x;
  const int64_t lo = (int64_t)r * a.N / a.G, hi = (int64_t)(r + 1) * a.N / a.G;
  int e[kRangeLoads];
#pragma unroll
  for (int u = 0; u < kRangeLoads; ++u) {
    const int i = u * kRangeThreads + tid;
    e[u] = i < a.M ? a.idx[i] : INT_MAX;
  }
  // own keys: counted per wave with ballots, a scan over the waves, then written in place
  int below = 0, own = 0;
#pragma unroll
  for (int u = 0; u < kRangeLoads; ++u) {
    const int i = u * kRangeThreads + tid;
    below += (i < a.M && e[u] < lo) ? 1 : 0;
    own += __popcll(__ballot(i < a.M && e[u] >= lo && e[u] < hi));
  }
  // one scan for both counts: the wave's own keys (from lane 0) above bit 16, the thread's
  // lower-range tasks below it (each total is at most 8192)
  int tot;
  const int ex = range_block_scan((l == 0 ? own << 16 : 0) + below, wsum, &tot);
  const int n = tot >> 16, n_below = tot & 0xFFFF;
  const int wbase = ex >> 16;
  if (n > kRangeCap) {
    if (tid == 0) a.range_heads[r] = -1;
    return;
  }
  for (int j = tid; j < n; j += kRangeThreads) rk[j] = 0;
  const uint64_t lt = lanemask_lt();
  int pos = __shfl(wbase, 0, kWave);
#pragma unroll
  for (int u = 0; u < kRangeLoads; ++u) {
    const int i = u * kRangeThreads + tid;
    const bool mine = i < a.M && e[u] >= lo && e[u] < hi;
    const uint64_t bal = __ballot(mine);
    if (mine) keys[pos + __popcll(bal & lt)] = ((uint64_t)(uint32_t)e[u] << 32) | (uint32_t)i;
    pos += __popcll(bal);
  }
  const int n8 = (n + 7) & ~7;
  if (tid < n8 - n) keys[n + tid] = ~0ull;
  __syncthreads();
  // place of key j: the number of smaller keys, counted by four threads over a quarter of the
  // keys each (eight per step, 16-byte broadcast reads) and added up in LDS
  constexpr int kParts = 4, kPerPass = kRangeThreads / kParts;
  const int part = tid / kPerPass;
  const int qlen = ((n8 / 8 + kParts - 1) / kParts) * 8;
  const int q0 = part * qlen < n8 ? part * qlen : n8;
  const int q1 = q0 + qlen < n8 ? q0 + qlen : n8;
  for (int j0 = 0; j0 < n; j0 += kPerPass) {
    const int j = j0 + tid % kPerPass;
    const uint64_t kj = j < n ? keys[j] : 0ull;
    int rank = 0;
    for (int q = q0; q < q1; q += 8) {
      const ulonglong2 k0 = *(const ulonglong2*)&keys[q];
      const ulonglong2 k1 = *(const ulonglong2*)&keys[q + 2];
      const ulonglong2 k2 = *(const ulonglong2*)&keys[q + 4];
      const ulonglong2 k3 = *(const ulonglong2*)&keys[q + 6];
      rank += (k0.x < kj) + (k0.y < kj) + (k1.x < kj) + (k1.y < kj) + (k2.x < kj) +
              (k2.y < kj) + (k3.x < kj) + (k3.y < kj);
    }
    if (j < n && rank > 0) atomicAdd(&rk[j], rank);
  }
  __syncthreads();
  for (int j = tid; j < n; j += kRangeThreads) sorted[rk[j]] = keys[j];
  __syncthreads();
  for (int j = tid; j < n; j += kRangeThreads) {
    const uint64_t k = sorted[j];
    a.perm[n_below + j] = (int32_t)(uint32_t)k;
    a.sorted[n_below + j] = (int32_t)(k >> 32);
  }
  // segment heads: thread t owns positions [t per, (t + 1) per)
  const int per = (n + kRangeThreads - 1) / kRangeThreads;
  const int j0 = tid * per;
  const int j1 = j0 + per < n ? j0 + per : n;
  int heads = 0;
  for (int j = j0; j < j1; ++j)
    heads += (j == 0 || (sorted[j] >> 32) != (sorted[j - 1] >> 32)) ? 1 : 0;
  int n_heads;
  int h = range_block_scan(heads, wsum, &n_heads);
  for (int j = j0; j < j1; ++j) {
    if (j == 0 || (sorted[j] >> 32) != (sorted[j - 1] >> 32)) {
      a.stage_act[n_below + h] = (int32_t)(sorted[j] >> 32);
      a.stage_off[n_below + h] = n_below + j;
      ++h;
    }
  }
  if (tid == 0) {
    a.range_base[r] = n_below;
    a.range_heads[r] = n_heads;
  }
}

__global__ __launch_bounds__(kSmallThreads) void schedule_small_kernel(SmallSched a) {
  __shared__ int cnt[kSmallWaves][kMaxRadix];
  __shared__ int dsum[kMaxRadix];
  __shared__ int wsum[kSmallWaves];
  // keys and task ids between radix passes, then the sorted keys; the bucket path's 64-bit keys
  __shared__ uint64_t sbuf[kSmallMax];
  int* skey = (int*)sbuf;
  int* sval = skey + kSmallMax;
  const int tid = threadIdx.x, l = lane_id(), w = tid >> 6;
  const int slice = (a.M + kSmallWaves - 1) / kSmallWaves;
  const int wbeg = w * slice;
  const int wend = wbeg + slice < a.M ? wbeg + slice : a.M;
  const uint64_t lt = lanemask_lt();
  if (a.G > 0) {
    // place the heads staged by schedule_ranges_kernel, unless a range overflowed
    const int hv = tid < a.G ? a.range_heads[tid] : 0;
    const int bv = tid < a.G ? a.range_base[tid] : 0;
    if (!__syncthreads_or(hv < 0)) {
      // workgroup r places range r's heads after the heads of ranges 0 .. r-1
      const int r = blockIdx.x;
      const int ex = wave_excl_scan_i32(hv);
      if (l == kWave - 1) wsum[w] = ex + hv;
      if (tid == r) {
        cnt[0][0] = hv;
        cnt[0][1] = bv;
        cnt[0][2] = ex;  // G <= 64: the scan within wave 0 is the whole scan
      }
      __syncthreads();
      int tot = 0;
      for (int ww = 0; ww < kSmallWaves; ++ww) tot += wsum[ww];
      const int nh = cnt[0][0], src = cnt[0][1], dst = cnt[0][2];
      for (int j = tid; j < nh; j += kSmallThreads) {
        const int va = a.stage_act[src + j], vo = a.stage_off[src + j];
        if (dst + j < a.cap) {
          a.active[dst + j] = va;
          a.offsets[dst + j] = vo;
        }
      }
      if (r != 0) return;
      if (tid == 0) {
        const int n = tot < a.cap ? tot : a.cap;
        *a.n_active = n;
        a.offsets[n] = a.M;
      }
      return;
    }
    if (blockIdx.x != 0) return;
  }
  // --- bucket path
  constexpr int kBuckets = 1024;  // = kSmallThreads: one bucket per thread in the scan
  constexpr int kBucketMax = 128;
  static_assert(kBuckets == kSmallThreads && kBuckets <= kMaxRadix, "bucket scan layout");
  int* bcount = cnt[0];
  int* bfill = cnt[1];
  int* bstart = cnt[2];
  int* bsorted = cnt[3];  // [kSmallMax] (rows 3 .. 10): expert of each sorted position
  uint64_t* bk = sbuf;  // [kSmallMax]
  static_assert(3 * kMaxRadix + kSmallMax <= kSmallWaves * kMaxRadix, "bucket arrays fit");
  const int hb = a.total_bits > 10 ? a.total_bits - 10 : 0;
  bcount[tid] = 0;
  bfill[tid] = 0;
  __syncthreads();
  uint64_t key64[kSmallRounds];
#pragma unroll
  for (int r = 0; r < kSmallRounds; ++r) {
    const int i = r * kSmallThreads + tid;
    key64[r] = ~0ull;
    if (i < a.M) {
      const uint32_t e = (uint32_t)a.idx[i];
      key64[r] = ((uint64_t)e << 32) | (uint32_t)i;
      atomicAdd(&bcount[(e >> hb) & (kBuckets - 1)], 1);
    }
  }
  __syncthreads();
  {
    const int c = bcount[tid];
    const int ex = wave_excl_scan_i32(c);
    int mx = c;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) mx = max(mx, __shfl_xor(mx, m, kWave));
    if (l == kWave - 1) wsum[w] = ex + c;
    if (l == 0) dsum[w] = mx;
    __syncthreads();
    int off = 0, big = 0;
    for (int ww = 0; ww < kSmallWaves; ++ww) {
      if (ww < w) off += wsum[ww];
      big = max(big, dsum[ww]);
    }
    bstart[tid] = off + ex;
    __syncthreads();
    if (big <= kBucketMax) {  // the same on every thread
#pragma unroll
      for (int r = 0; r < kSmallRounds; ++r) {
        const int i = r * kSmallThreads + tid;
        if (i < a.M) {
          const int b = (int)((uint32_t)(key64[r] >> 32) >> hb) & (kBuckets - 1);
          bk[bstart[b] + atomicAdd(&bfill[b], 1)] = key64[r];
        }
      }
      __syncthreads();
      // taken in bucket order, so the lanes of a wave mostly scan the same bucket (broadcast
      // reads); the keys then move to their final places in LDS
      int fpos[kSmallRounds];
#pragma unroll
      for (int r = 0; r < kSmallRounds; ++r) {
        const int i = r * kSmallThreads + tid;
        fpos[r] = -1;
        if (i < a.M) {
          const uint64_t key = bk[i];
          key64[r] = key;
          const int b = (int)((uint32_t)(key >> 32) >> hb) & (kBuckets - 1);
          const int b0 = bstart[b], n = bcount[b];
          int rank = 0;
          for (int q = 0; q < n; ++q) rank += bk[b0 + q] < key ? 1 : 0;
          fpos[r] = b0 + rank;
        }
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < kSmallRounds; ++r)
        if (fpos[r] >= 0) bk[fpos[r]] = key64[r];
      __syncthreads();
      small_out_sorted(a, bk, bsorted, wsum);
      return;
    }
  }
  // --- radix path (a crowded bucket)
  int shift = 0;
  for (int ps = 0; ps < a.passes; ++ps) {
    const bool last = ps == a.passes - 1;
    int bits = a.total_bits - shift;
    if (bits > a.per) bits = a.per;
    if (bits < 1) bits = 1;
    const int radix = 1 << bits;
    const uint32_t mask = (uint32_t)radix - 1u;
    for (int i = tid; i < kSmallWaves * kMaxRadix; i += kSmallThreads) (&cnt[0][0])[i] = 0;
    int key[kSmallRounds], val[kSmallRounds], rank[kSmallRounds];
#pragma unroll
    for (int r = 0; r < kSmallRounds; ++r) {
      const int i = wbeg + r * kWave + l;
      const bool valid = i < wend;
      key[r] = valid ? (ps == 0 ? a.idx[i] : skey[i]) : 0;
      val[r] = valid ? (ps == 0 ? i : sval[i]) : 0;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSmallRounds; ++r) {
      const int i = wbeg + r * kWave + l;
      const bool valid = i < wend;
      const uint32_t d = ((uint32_t)key[r] >> shift) & mask;
      uint64_t peers = __ballot(valid);
      for (int b = 0; b < bits; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t bal = __ballot(bit);
        peers &= bit ? bal : ~bal;
      }
      const int before = __popcll(peers & lt);
      const int run = valid ? cnt[w][d] : 0;
      wave_lds_sync();
      if (valid && before == 0) cnt[w][d] = run + __popcll(peers);
      wave_lds_sync();
      rank[r] = run + before;
    }
    __syncthreads();
    // digit totals, their exclusive scan, then (digit, wave) offsets
    for (int d = tid; d < radix; d += kSmallThreads) {
      int t = 0;
      for (int ww = 0; ww < kSmallWaves; ++ww) t += cnt[ww][d];
      dsum[d] = t;
    }
    __syncthreads();
    {
      // exclusive scan of the digit totals: one digit per thread (radix <= 1024 threads)
      const int v = tid < radix ? dsum[tid] : 0;
      const int ex = wave_excl_scan_i32(v);
      if (l == kWave - 1) wsum[w] = ex + v;
      __syncthreads();
      int off = 0;
      for (int ww = 0; ww < w; ++ww) off += wsum[ww];
      if (tid < radix) dsum[tid] = off + ex;
    }
    __syncthreads();
    for (int d = tid; d < radix; d += kSmallThreads) {
      int run = dsum[d];
      for (int ww = 0; ww < kSmallWaves; ++ww) {
        const int c = cnt[ww][d];
        cnt[ww][d] = run;
        run += c;
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSmallRounds; ++r) {
      const int i = wbeg + r * kWave + l;
      if (i < wend) {
        const uint32_t d = ((uint32_t)key[r] >> shift) & mask;
        const int pos = cnt[w][d] + rank[r];
        skey[pos] = key[r];
        sval[pos] = val[r];
        if (last) {
          a.sorted[pos] = key[r];
          a.perm[pos] = val[r];
        }
      }
    }
    __syncthreads();
    shift += bits;
  }
  small_heads(a, skey, wsum);
}

hipError_t launch_fill_i32(int32_t* dst, int64_t n, int32_t value, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, st, dst, n, value);
  return hipGetLastError();
}

namespace {

int64_t partial_count(int64_t M) {
  const int64_t tiles = (M + kTile - 1) / kTile;
  const int64_t hist = (int64_t)kMaxRadix * (tiles > 0 ? tiles : 1);
  return (std::max<int64_t>(hist, M) + kTile - 1) / kTile + 1;
}

// Scan partials of a schedule: the sort's scans over M tasks, and a scan over the N experts.
int64_t sched_partial_count(int64_t M, int64_t N) {
  return std::max<int64_t>(partial_count(M), (N + kTile - 1) / kTile + 1);
}

struct SortBuffers {
  int32_t *k0, *v0, *k1, *v1, *hist, *partial;
};

// Stable LSD radix sort of the task ids 0 .. M-1 by keys[] (all below 2^total_bits), in the
// fewest passes of at most 10 bits. The sorted task ids go to ids_out; *keys_out points to the
// sorted keys (one of the ping-pong buffers).
hipError_t radix_sort_tasks(const int32_t* keys, int64_t M, int total_bits, int32_t* ids_out,
                            const SortBuffers& b, const int32_t** keys_out, hipStream_t st) {
  const int passes = total_bits == 0 ? 1 : (total_bits + kMaxDigitBits - 1) / kMaxDigitBits;
  const int per = total_bits == 0 ? 1 : (total_bits + passes - 1) / passes;
  const int num_tiles = (int)((M + kTile - 1) / kTile);
  const int32_t* kin = keys;
  const int32_t* vin = nullptr;
  int shift = 0;
  for (int ps = 0; ps < passes; ++ps) {
    const bool last = ps == passes - 1;
    const int bits = std::min(per, std::max(1, total_bits - shift));
    RadixPass p;
    p.keys_in = kin;
    p.vals_in = vin;
    p.keys_out = (ps & 1) ? b.k1 : b.k0;
    p.vals_out = last ? ids_out : ((ps & 1) ? b.v1 : b.v0);
    p.hist = b.hist;
    p.n = M;
    p.shift = shift;
    p.bits = bits;
    p.num_tiles = num_tiles;
    hipLaunchKernelGGL(radix_upsweep_kernel, dim3(num_tiles), dim3(kThreads), 0, st, p);
    const int64_t hn = (int64_t)(1 << bits) * num_tiles;
    hipError_t e = device_scan(ArrayVal{b.hist, hn}, EmitScan{b.hist, hn}, hn, b.partial, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(radix_downsweep_kernel, dim3(num_tiles), dim3(kThreads), 0, st, p);
    kin = p.keys_out;
    vin = p.vals_out;
    shift += bits;
  }
  *keys_out = kin;
  return hipGetLastError();
}

}  // namespace

size_t schedule_ws_bytes(int64_t M, int64_t N) {
  const int64_t tiles = (M + kTile - 1) / kTile;
  const int64_t hist = (int64_t)kMaxRadix * (tiles > 0 ? tiles : 1);
  size_t b = 0;
  b += 4 * align_up((size_t)M * 4);               // keys/values ping-pong
  b += align_up((size_t)hist * 4);                // histogram
  b += align_up((size_t)sched_partial_count(M, N) * 4);  // scan partials
  b += align_up((size_t)N * 4);                   // expert -> rank in the active list (B > 1)
  b += align_up((size_t)M * 4);                   // group key of every task (B > 1)
  return b;
}

int group_key_bits(const Shape& s) {
  const int64_t cap = std::min<int64_t>(s.M, s.N);
  const int gb = digit_bits_total((cap + s.B - 1) / s.B);
  return gb > 0 ? gb : 1;
}

hipError_t launch_schedule(const Shape& s, const int32_t* idx, int32_t* perm, int32_t* active,
                           int32_t* active_offsets, int32_t* n_active, int32_t* dense_offsets,
                           void* ws, const int32_t** sorted_keys, hipStream_t st,
                           const int32_t** group_keys) {
  const int64_t M = s.M;
  const int64_t tiles = (M + kTile - 1) / kTile;
  char* w = (char*)ws;
  SortBuffers b;
  b.k0 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.v0 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.k1 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.v1 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.hist = (int32_t*)w; w += align_up((size_t)kMaxRadix * (tiles > 0 ? tiles : 1) * 4);
  b.partial = (int32_t*)w; w += align_up((size_t)sched_partial_count(M, s.N) * 4);
  int32_t* rank = (int32_t*)w; w += align_up((size_t)s.N * 4);
  int32_t* gkey = (int32_t*)w;
  const int64_t cap64 = std::min<int64_t>(M, s.N);
  const int32_t cap = (int32_t)cap64;

  // Digit widths: the fewest passes of at most 10 bits, spread evenly.
  const int total_bits = digit_bits_total(s.N);
  if (M <= kSmallMax) {
    const int passes = total_bits == 0 ? 1 : (total_bits + kMaxDigitBits - 1) / kMaxDigitBits;
    const int per = total_bits == 0 ? 1 : (total_bits + passes - 1) / passes;
    SmallSched a;
    a.idx = idx;
    a.sorted = b.k0;
    a.perm = perm;
    a.active = active;
    a.offsets = active_offsets;
    a.n_active = n_active;
    a.M = (int)M;
    a.cap = cap;
    a.passes = passes;
    a.per = per;
    a.total_bits = total_bits;
    a.G = 0;
    if (M > kRangeMinTasks) {
      RangeSched r;
      r.idx = idx;
      r.sorted = b.k0;
      r.perm = perm;
      r.stage_act = b.v0;
      r.stage_off = b.k1;
      r.G = (int)((M + kRangeTasks - 1) / kRangeTasks);
      r.range_base = b.v1;
      r.range_heads = b.v1 + r.G;
      r.N = s.N;
      r.M = (int)M;
      hipLaunchKernelGGL(schedule_ranges_kernel, dim3(r.G), dim3(kRangeThreads), 0, st, r);
      a.stage_act = r.stage_act;
      a.stage_off = r.stage_off;
      a.range_base = r.range_base;
      a.range_heads = r.range_heads;
      a.G = r.G;
    }
    // with ranges: one workgroup per range places its heads; only workgroup 0 sorts when a
    // range overflowed
    hipLaunchKernelGGL(schedule_small_kernel, dim3(a.G > 0 ? a.G : 1), dim3(kSmallThreads), 0, st,
                       a);
    *sorted_keys = b.k0;
  } else {
    const int32_t* sk = nullptr;
    hipError_t e = radix_sort_tasks(idx, M, total_bits, perm, b, &sk, st);
    if (e != hipSuccess) return e;
    *sorted_keys = sk;
    e = device_scan(HeadFlag{sk, M},
                    EmitSegments{sk, active, active_offsets, n_active, cap, (int32_t)M}, M,
                    b.partial, st);
    if (e != hipSuccess) return e;
  }
  if (dense_offsets) {
    const int64_t n = s.N + 1;
    hipLaunchKernelGGL(dense_offsets_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, st, (const int32_t*)active,
                       (const int32_t*)active_offsets, (const int32_t*)n_active, dense_offsets,
                       s.N);
  }
  if (s.B > 1) {
    // Groups of B active experts: order the tasks by (rank / B, task id).
    hipLaunchKernelGGL(rank_fill_kernel, dim3((unsigned)((cap64 + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, st, (const int32_t*)active, (const int32_t*)n_active,
                       rank, cap64, s.N);
    const int gb = group_key_bits(s);
    hipLaunchKernelGGL(group_key_kernel, dim3(key_blocks(M)), dim3(kThreads), 0, st, idx,
                       (const int32_t*)rank, gkey, M, s.N, s.B, div_magic((uint32_t)s.B), gb);
    const int32_t* gk = nullptr;
    hipError_t e = radix_sort_tasks(gkey, M, gb, perm, b, &gk, st);
    if (e != hipSuccess) return e;
    *sorted_keys = nullptr;
    if (group_keys) *group_keys = gk;
  }
  return hipGetLastError();
}


// The grouped layer's schedule without the sort by expert: the active list only needs to know
// which experts have tasks, so a bitmap of them (mark_experts_kernel) and one scan over its words
// give the ascending active list and every expert's rank; the group keys and the stable sort by
// group key then run as in launch_schedule. Same workspace: the bitmap and its prefix take the
// rank array's place.
bool group_schedule_fits(const Shape& s) { return (s.N + 31) / 32 <= kMapWords; }

hipError_t launch_group_schedule(const Shape& s, const int32_t* idx, int32_t* perm,
                                 int32_t* active, int32_t* n_active, void* ws,
                                 const int32_t** group_keys, hipStream_t st) {
  if (!group_schedule_fits(s)) return hipErrorInvalidValue;
  const int64_t M = s.M;
  const int64_t tiles = (M + kTile - 1) / kTile;
  char* w = (char*)ws;
  SortBuffers b;
  b.k0 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.v0 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.k1 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.v1 = (int32_t*)w; w += align_up((size_t)M * 4);
  b.hist = (int32_t*)w; w += align_up((size_t)kMaxRadix * (tiles > 0 ? tiles : 1) * 4);
  b.partial = (int32_t*)w; w += align_up((size_t)sched_partial_count(M, s.N) * 4);
  // 2 * words <= max(64, N) ints: inside the rank array
  const int words = (int)((s.N + 31) / 32);
  uint32_t* bits = (uint32_t*)w;
  int32_t* prefix = (int32_t*)w + words;
  w += align_up((size_t)s.N * 4);
  int32_t* gkey = (int32_t*)w;
  const int32_t cap = (int32_t)std::min<int64_t>(M, s.N);
  const int64_t rounds = (M + kMapChunk - 1) / kMapChunk;
  const unsigned grid = (unsigned)std::min<int64_t>(rounds, 512);
  hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)((words + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, st, (int32_t*)bits, (int64_t)words, 0);
  hipLaunchKernelGGL(mark_experts_kernel, dim3(grid), dim3(kMapThreads), (size_t)words * 4, st,
                     idx, bits, M, s.N, words);
  hipError_t e = device_scan(PopWord{bits, words}, EmitPrefix{prefix, n_active, words, cap},
                             words, b.partial, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(list_active_kernel, dim3((unsigned)((s.N + kThreads - 1) / kThreads)),
                     dim3(kThreads), 0, st, (const uint32_t*)bits, (const int32_t*)prefix, active,
                     s.N, cap);
  const int gb = group_key_bits(s);
  hipLaunchKernelGGL(group_key_map_kernel, dim3(grid), dim3(kMapThreads), (size_t)words * 8, st,
                     idx, (const uint32_t*)bits, (const int32_t*)prefix, gkey, M, s.N, words,
                     s.B, div_magic((uint32_t)s.B), gb);
  return radix_sort_tasks(gkey, M, gb, perm, b, group_keys, st);
}

int64_t group_count_bound(const Shape& s) {
  const int64_t cap = std::min<int64_t>(s.M, s.N);
  return (cap + s.B - 1) / s.B;
}

size_t group_plan_ws_bytes(const Shape& s) {
  const int64_t G = group_count_bound(s);
  size_t b = 0;
  b += align_up((size_t)s.N * 4);                  // rank (caller's schedule only)
  b += align_up((size_t)s.M * 4);                  // packed keys (caller's schedule only)
  b += align_up((size_t)s.M * 4);                  // slot_token
  b += align_up((size_t)(s.M + 1) * 4);            // slot_off
  b += 2 * align_up((size_t)(G + 1) * 4);          // grp_slot, grp_tile
  b += align_up((size_t)partial_count(s.M) * 4);   // scan partials
  b += 256;                                        // counters
  return b;
}

hipError_t launch_group_plan(const Shape& s, const int32_t* perm, const int32_t* n_active,
                             const int32_t* sorted_group_keys, const int32_t* idx,
                             const int32_t* active, void* ws, GroupPlan* plan,
                             hipStream_t st) {
  const int64_t M = s.M;
  const int64_t G = group_count_bound(s);
  const int64_t cap = std::min<int64_t>(M, s.N);
  char* w = (char*)ws;
  int32_t* rank = (int32_t*)w; w += align_up((size_t)s.N * 4);
  int32_t* keys = (int32_t*)w; w += align_up((size_t)M * 4);
  plan->slot_token = (int32_t*)w; w += align_up((size_t)M * 4);
  plan->slot_off = (int32_t*)w; w += align_up((size_t)(M + 1) * 4);
  plan->grp_slot = (int32_t*)w; w += align_up((size_t)(G + 1) * 4);
  plan->grp_tile = (int32_t*)w; w += align_up((size_t)(G + 1) * 4);
  int32_t* partial = (int32_t*)w; w += align_up((size_t)partial_count(M) * 4);
  plan->counters = (int32_t*)w;
  plan->G = G;
  plan->gbits = group_key_bits(s);
  if (sorted_group_keys) {
    plan->key = sorted_group_keys;
  } else {
    hipLaunchKernelGGL(rank_fill_kernel, dim3((unsigned)((cap + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, st, active, n_active, rank, cap, s.N);
    hipLaunchKernelGGL(position_key_kernel, dim3(key_blocks(M)), dim3(kThreads), 0, st, perm,
                       idx, (const int32_t*)rank, keys, M, s.N, s.B, div_magic((uint32_t)s.B),
                       plan->gbits);
    plan->key = keys;
  }
  const SlotHead head{perm, plan->key, M, (1u << plan->gbits) - 1u,
                      div_magic((uint32_t)s.hk)};
  const int nb = (int)((M + kTile - 1) / kTile);
  hipLaunchKernelGGL(scan_reduce_kernel<SlotHead>, dim3(nb), dim3(kThreads), 0, st, head, M,
                     partial);
  hipLaunchKernelGGL(slot_heads_down_kernel, dim3(nb), dim3(kThreads), 0, st,
                     EmitSlots{head, n_active, G, s.B, plan->slot_token, plan->slot_off,
                               plan->grp_slot, plan->counters},
                     (const int32_t*)partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return device_scan(GroupTiles{plan->grp_slot, n_active, G, s.B, grouped_tile_experts(s.B)},
                     EmitTiles{plan->grp_tile, G + 1, plan->counters}, G + 1, partial, st);
}

// ---------------------------------------------------------------- slots by token
// The second product of Eq. 14 per group leaves one partial row per (group, token) slot; the
// token's output is the sum of its slots' rows in group order. The slots are listed group by
// group (tokens ascending inside a group), so a stable sort of the slot ids by token gives every
// token's slots as one run in group order. Slot ids n_slots <= s < n (unused entries) get the
// key T and sort last.

namespace {

__global__ __launch_bounds__(kThreads) void slot_key_kernel(const int32_t* __restrict__ slot_token,
                                                          const int32_t* __restrict__ counters,
                                                          int32_t* __restrict__ key, int64_t n,
                                                          int32_t T) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) key[i] = i < counters[0] ? slot_token[i] : T;
}

// tok_start[t] = first place of token t in the sorted order (-1 when t has no slot).
__global__ __launch_bounds__(kThreads) void token_start_kernel(const int32_t* __restrict__ sk,
                                                             int32_t* __restrict__ tok_start,
                                                             int64_t n, int32_t T) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const int32_t k = sk[i];
  if (k < T && (i == 0 || sk[i - 1] != k)) tok_start[k] = (int32_t)i;
}

}  // namespace

size_t slot_sort_ws_bytes(int64_t n, int64_t T) {
  const int64_t tiles = (n + kTile - 1) / kTile;
  const int64_t hist = (int64_t)kMaxRadix * (tiles > 0 ? tiles : 1);
  size_t b = 0;
  b += 6 * align_up((size_t)n * 4);             // keys, ping-pong keys/values, sorted ids
  b += align_up((size_t)hist * 4);              // histogram
  b += align_up((size_t)partial_count(n) * 4);  // scan partials
  b += align_up((size_t)(T + 1) * 4);           // token starts
  return b;
}

hipError_t launch_slot_sort(const GroupPlan& plan, int64_t n, int64_t T, void* ws,
                            SlotOrder* out, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  char* w = (char*)ws;
  int32_t* key = (int32_t*)w; w += align_up((size_t)n * 4);
  SortBuffers b;
  b.k0 = (int32_t*)w; w += align_up((size_t)n * 4);
  b.v0 = (int32_t*)w; w += align_up((size_t)n * 4);
  b.k1 = (int32_t*)w; w += align_up((size_t)n * 4);
  b.v1 = (int32_t*)w; w += align_up((size_t)n * 4);
  int32_t* ids = (int32_t*)w; w += align_up((size_t)n * 4);
  const int64_t tiles = (n + kTile - 1) / kTile;
  b.hist = (int32_t*)w; w += align_up((size_t)kMaxRadix * (tiles > 0 ? tiles : 1) * 4);
  b.partial = (int32_t*)w; w += align_up((size_t)partial_count(n) * 4);
  int32_t* tok_start = (int32_t*)w;
  const unsigned grid = (unsigned)((n + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(slot_key_kernel, dim3(grid), dim3(kThreads), 0, st, plan.slot_token,
                     plan.counters, key, n, (int32_t)T);
  int bits = 1;
  while ((1ll << bits) <= T) ++bits;  // keys 0 .. T
  const int32_t* sk = nullptr;
  hipError_t e = radix_sort_tasks(key, n, bits, ids, b, &sk, st);
  if (e != hipSuccess) return e;
  if ((e = launch_fill_i32(tok_start, T, -1, st)) != hipSuccess) return e;
  hipLaunchKernelGGL(token_start_kernel, dim3(grid), dim3(kThreads), 0, st, sk, tok_start, n,
                     (int32_t)T);
  out->slots = ids;
  out->tokens = sk;
  out->tok_start = tok_start;
  return hipGetLastError();
}

}  // namespace omnimoe
