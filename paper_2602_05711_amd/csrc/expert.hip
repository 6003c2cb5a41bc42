// Per-expert vector compute (Eq. 4, 7, 14).
//
// expert_dot: expert-major. The schedule's sorted positions are cut into ranges of about 8, 16
// or 64 tasks, each starting at an expert boundary (a range only starts inside an expert's run
// when the run is longer than the range, so very hot experts are shared out); each XCD takes a
// contiguous share of the ranges. One wavefront walks its range run by run: it loads the
// expert's u row once (16-byte loads with the non-temporal hint, every lane a slice),
// then for up to four of the run's tasks at a time loads the token rows, forms the dot
// products in fp32, and writes a[p] = g_p * act(x_t . u_e) into the token-major slot p.
//
// slot_dot: the same a[p] in slot order, without a schedule, where the expert-major order saves
// no memory traffic (a decode step, few tasks per expert, tables that stay in the MALL).
//
// accumulate: token-major, one wavefront per token. The token's H*K slots are read in
// (head, k) order, their v rows are fetched eight at a time and y_t += a[p] * v_e is summed in
// slot order in fp32. The order is fixed, so y is the same on every run; no atomics are used.
// With too few tokens to fill the chip, a token's row is split over column ranges and its slots
// over the waves of a workgroup, whose partial rows are added in wave order.
//
// scatter_contrib / reduce_contrib: the output stage in expert-major order (v read once per
// expert run) through per-task fp32 contribution rows and a token-major sum of them.
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

struct DotArgs {
  const void* x;
  const void* u;
  const int32_t* idx;
  const float* gates;
  const int32_t* perm;
  const int32_t* sk;  // expert of each sorted position, or NULL
  float* a;
  int64_t M;
  int64_t N;
  int d;
  int hk;
  int act;
  int nchunks;  // 16-byte chunks per row
  int range;    // nominal tasks per wave (power of two <= 64)
};

struct AccArgs {
  const void* v;
  const int32_t* idx;
  const float* a;
  float* y;
  int64_t T;
  int64_t N;
  int d;
  int hk;
  int nchunks;
  int splits;  // waves per token; wave c of a token owns chunk rows [c CPL, (c + 1) CPL)
};

// Ids and task numbers are clamped into range, so malformed inputs cannot address memory
// outside the tables (their results are then meaningless).
__device__ __forceinline__ int clamp_i(int v, int64_t n) {
  return v < 0 ? 0 : (v >= n ? (int)(n - 1) : v);
}

__device__ __forceinline__ int task_at(const DotArgs& a, int64_t pos) {
  return clamp_i(a.perm[pos], a.M);
}

__device__ __forceinline__ int key_at(const DotArgs& a, int64_t pos) {
  return clamp_i(a.sk ? a.sk[pos] : a.idx[task_at(a, pos)], a.N);
}

// First position of the wave range starting near lo: the first expert boundary in
// [lo, lo + range), or lo + range when that window lies inside one expert's run.
__device__ int64_t range_start(const DotArgs& a, int64_t lo) {
  if (lo >= a.M) return a.M;
  const int l = lane_id();
  const int64_t pos = lo + l;
  const bool in = l < a.range && pos < a.M;
  const int key = in ? key_at(a, pos) : -1;
  const int before = lo > 0 ? key_at(a, lo - 1) : -1;
  int prev = __shfl_up(key, 1, kWave);
  if (l == 0) prev = before;
  const uint64_t heads = __ballot(in && key != prev);
  if (heads) return lo + (__ffsll((unsigned long long)heads) - 1);
  const int64_t nx = lo + a.range;
  return nx < a.M ? nx : a.M;
}

template <int CPL>
__device__ __forceinline__ void load_row(uint4 (&r)[CPL], const uint4* base, const bool (&cv)[CPL]) {
  const int l = lane_id();
#pragma unroll
  for (int q = 0; q < CPL; ++q) r[q] = cv[q] ? base[l + kWave * q] : make_uint4(0, 0, 0, 0);
}

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// load_row with the non-temporal hint: for rows read once (an expert's u row), so that they
// do not push out of L2 the token rows that are read again.
template <int CPL>
__device__ __forceinline__ void load_row_nt(uint4 (&r)[CPL], const uint4* base,
                                            const bool (&cv)[CPL]) {
  const int l = lane_id();
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    if (cv[q]) {
      const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)(base + l + kWave * q));
      r[q] = make_uint4(v.x, v.y, v.z, v.w);
    } else {
      r[q] = make_uint4(0, 0, 0, 0);
    }
  }
}

// Positions are taken G at a time (four for rows up to 4096 bf16 values). Slot i holds position j0 + i: its token row is loaded,
// and its expert's u row is loaded only when that expert differs from the previous position's
// (otherwise the previous slot's registers are copied), so each run of an expert reads u once.
// Every load of a group is issued before the first copy: a copy waits for the row it copies,
// and a wait placed between the slots' loads would leave one slot's rows in flight at a time.
// FULL: the row is exactly CPL * 64 chunks, so the loads need no per-chunk guard (guarded
// loads also make the compiler wait for every outstanding load at each copy).
template <int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(256) void expert_dot_kernel(DotArgs a) {
  constexpr int G = CPL >= 16 ? 1 : (CPL >= 8 ? 2 : 4);
  const int l = lane_id();
  // Workgroup b runs on XCD b % 8; each XCD takes a contiguous share of the sorted positions,
  // so the token rows that recur within a stretch of the expert order (a token's experts in
  // one grid row are neighbours there) are fetched into that XCD's L2 once.
  const int64_t nb = gridDim.x, per_xcd = nb / 8, extra = nb % 8, xcd = blockIdx.x % 8;
  const int64_t blk = xcd * per_xcd + (xcd < extra ? xcd : extra) + blockIdx.x / 8;
  const int64_t wave = blk * 4 + (threadIdx.x >> 6);
  const int64_t s = range_start(a, wave * a.range);
  const int64_t e = range_start(a, (wave + 1) * a.range);
  if (s >= e) return;
  const uint4* X = (const uint4*)a.x;
  const uint4* U = (const uint4*)a.u;
  const int64_t row_chunks = a.nchunks;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = FULL || (l + kWave * q) < a.nchunks;

  // token of a task: p / (H K), a shift when H K is a power of two (a 32-bit division is some
  // fifteen scalar instructions, issued for every task)
  const int hk_shift = (a.hk & (a.hk - 1)) == 0 ? __builtin_ctz((unsigned)a.hk) : -1;
  auto token_of = [&](int p) { return hk_shift >= 0 ? p >> hk_shift : p / a.hk; };

  int prev = -1;    // expert whose u row sits in ur[G - 1]
  uint4 ur[G][CPL];
  uint4 xr[G][CPL];
#pragma unroll
  for (int i = 0; i < G; ++i)
#pragma unroll
    for (int q = 0; q < CPL; ++q) ur[i][q] = make_uint4(0, 0, 0, 0);
  for (int64_t b = s; b < e; b += kWave) {
    const int64_t pos = b + l;
    const bool v = pos < e;
    const int key = v ? key_at(a, pos) : -1;
    const int p = v ? task_at(a, pos) : 0;
    const float g = v ? a.gates[p] : 0.0f;
    const int cnt = (int)((e - b) < kWave ? (e - b) : kWave);
    for (int j0 = 0; j0 < cnt; j0 += G) {
      int ej[G], pj[G];
      float gj[G];
#pragma unroll
      for (int i = 0; i < G; ++i) {
        const int jj = (j0 + i < cnt) ? j0 + i : cnt - 1;
        ej[i] = readlane_i32(key, jj);
        pj[i] = readlane_i32(p, jj);
        gj[i] = readlane_f32(g, jj);
      }
      // the first slot takes the carried row before a load of this group can replace it
      if (G > 1 && ej[0] == prev) {
#pragma unroll
        for (int q = 0; q < CPL; ++q) ur[0][q] = ur[G - 1][q];
      }
#pragma unroll
      for (int i = 0; i < G; ++i)
        if (j0 + i < cnt) load_row<CPL>(xr[i], X + (int64_t)token_of(pj[i]) * row_chunks, cv);
#pragma unroll
      for (int i = 0; i < G; ++i) {
        const int before = (i == 0) ? prev : ej[i - 1];
        if (j0 + i < cnt && ej[i] != before)
          load_row_nt<CPL>(ur[i], U + (int64_t)ej[i] * row_chunks, cv);
      }
      // slots that repeat their predecessor's expert share its row (in slot order, so that a
      // run of several slots copies along)
#pragma unroll
      for (int i = 1; i < G; ++i) {
        if (j0 + i < cnt && ej[i] == ej[i - 1]) {
#pragma unroll
          for (int q = 0; q < CPL; ++q) ur[i][q] = ur[i - 1][q];
        }
      }
      float h[G];
#pragma unroll
      for (int i = 0; i < G; ++i) {
        float acc = 0.0f;
#pragma unroll
        for (int q = 0; q < CPL; ++q) acc = chunk_dot<BF16>(ur[i][q], xr[i][q], acc);
        h[i] = acc;
      }
      // lane i finishes task j0 + i: one activation for the group instead of one per task
      float hv = 0.0f, gv = 0.0f;
      int pv = 0;
#pragma unroll
      for (int i = 0; i < G; ++i) {
        if (j0 + i < cnt) {
          const float hs = wave_sum_uniform(h[i]);
          if (l == i) {
            hv = hs;
            gv = gj[i];
            pv = pj[i];
          }
        }
      }
      if (l < G && j0 + l < cnt) a.a[pv] = gv * activation(a.act, hv);
      // The last filled slot's expert carries into the next group.
      const int last = (cnt - j0 < G ? cnt - j0 : G) - 1;
#pragma unroll
      for (int i = 0; i < G - 1; ++i)
        if (i == last) {
#pragma unroll
          for (int q = 0; q < CPL; ++q) ur[G - 1][q] = ur[i][q];
        }
      prev = ej[last];
    }
  }
}

// The batch's v row loads are guarded (a slot past the end loads nothing), and with guarded loads
// the compiler waits for each row before issuing the next, so a wave fetches its rows one after
// another. Unguarded loads with all eight rows in flight (as in accumulate_slots_kernel) were
// slower here at the training shape, 1.44 -> 1.50 ms, and so were two or four rows in flight.
template <int CPL, bool BF16>
__global__ __launch_bounds__(256) void accumulate_kernel(AccArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int UNROLL = CPL >= 16 ? 2 : (CPL >= 8 ? 4 : 8);
  const int l = lane_id();
  const uint4* V = (const uint4*)a.v;
  const int64_t row_chunks = a.nchunks;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t wt = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wt < a.T * a.splits;
       wt += stride) {
    const int64_t t = wt / a.splits;
    const int cbase = (int)(wt % a.splits) * CPL * kWave;  // first chunk of this wave
    bool cvalid[CPL];
#pragma unroll
    for (int q = 0; q < CPL; ++q) cvalid[q] = (cbase + l + kWave * q) < a.nchunks;
    float acc[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = 0.0f;
    for (int sb = 0; sb < a.hk; sb += kWave) {
      const int sl = sb + l;
      const bool valid = sl < a.hk;
      const int ev = valid ? clamp_i(a.idx[t * a.hk + sl], a.N) : 0;
      const float av = valid ? a.a[t * a.hk + sl] : 0.0f;
      const int n = a.hk - sb < kWave ? a.hk - sb : kWave;
      for (int j = 0; j < n; j += UNROLL) {
        uint4 vr[UNROLL][CPL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
          if (j + u < n) {
            const int e = readlane_i32(ev, j + u);
            const uint4* vb = V + (int64_t)e * row_chunks + cbase;
#pragma unroll
            for (int q = 0; q < CPL; ++q)
              vr[u][q] = cvalid[q] ? vb[l + kWave * q] : make_uint4(0, 0, 0, 0);
          }
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
          if (j + u < n) {
            const float w = readlane_f32(av, j + u);
#pragma unroll
            for (int q = 0; q < CPL; ++q) {
              const uint4 c = vr[u][q];
              if constexpr (BF16) {
                acc[q][0] = fmaf(w, bf16_lo(c.x), acc[q][0]);
                acc[q][1] = fmaf(w, bf16_hi(c.x), acc[q][1]);
                acc[q][2] = fmaf(w, bf16_lo(c.y), acc[q][2]);
                acc[q][3] = fmaf(w, bf16_hi(c.y), acc[q][3]);
                acc[q][4] = fmaf(w, bf16_lo(c.z), acc[q][4]);
                acc[q][5] = fmaf(w, bf16_hi(c.z), acc[q][5]);
                acc[q][6] = fmaf(w, bf16_lo(c.w), acc[q][6]);
                acc[q][7] = fmaf(w, bf16_hi(c.w), acc[q][7]);
              } else {
                acc[q][0] = fmaf(w, __uint_as_float(c.x), acc[q][0]);
                acc[q][1] = fmaf(w, __uint_as_float(c.y), acc[q][1]);
                acc[q][2] = fmaf(w, __uint_as_float(c.z), acc[q][2]);
                acc[q][3] = fmaf(w, __uint_as_float(c.w), acc[q][3]);
              }
            }
          }
        }
      }
    }
    // y is written once and not read back here: non-temporal stores keep it out of the caches
    // the v gathers use.
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    f32x4_t* yt = (f32x4_t*)(a.y + t * a.d);
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!cvalid[q]) continue;
      const int c = cbase + l + kWave * q;
#pragma unroll
      for (int k = 0; k < EPC; k += 4) {
        const f32x4_t o = {acc[q][k], acc[q][k + 1], acc[q][k + 2], acc[q][k + 3]};
        __builtin_nontemporal_store(o, &yt[(c * EPC + k) / 4]);
      }
    }
  }
}

// Few tokens: a workgroup of W waves owns one (token, column split); wave w takes the w-th
// of W equal runs of the token's slots, so that all of a wave's v rows are in flight at once.
// The waves' partial rows go through LDS (in y order) and are added in wave order, so the
// per-element order is fixed. The row loads of a batch carry no guard (FULL: the column split
// is exactly CPL * 64 chunks; past the wave's last slot its row is loaded again), so the
// compiler issues them all before the first wait: 7.1 -> 6.5 us for the routed sum of one
// decoded token.
template <int W, int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(64 * W) void accumulate_slots_kernel(AccArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int UNROLL = CPL >= 16 ? 2 : (CPL >= 8 ? 4 : 8);
  constexpr int ROW = CPL * EPC * kWave;  // floats of one wave's partial row
  __shared__ __attribute__((aligned(16))) float part[W][ROW];
  // the wave number through an SGPR, so that the slot bounds and branches below are scalar
  const int l = lane_id(), w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint4* V = (const uint4*)a.v;
  const int64_t row_chunks = a.nchunks;
  const int per = (a.hk + W - 1) / W;
  const int s_lo = w * per < a.hk ? w * per : a.hk;
  const int s_hi = s_lo + per < a.hk ? s_lo + per : a.hk;
  for (int64_t u = blockIdx.x; u < a.T * a.splits; u += gridDim.x) {
    const int64_t t = u / a.splits;
    const int cbase = (int)(u % a.splits) * CPL * kWave;
    bool cvalid[CPL];
#pragma unroll
    for (int q = 0; q < CPL; ++q) cvalid[q] = FULL || (cbase + l + kWave * q) < a.nchunks;
    float acc[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = 0.0f;
    for (int sb = s_lo; sb < s_hi; sb += kWave) {
      const int sl = sb + l;
      const bool valid = sl < s_hi;
      const int ev = valid ? clamp_i(a.idx[t * a.hk + sl], a.N) : 0;
      const float av = valid ? a.a[t * a.hk + sl] : 0.0f;
      const int n = s_hi - sb < kWave ? s_hi - sb : kWave;
      for (int j = 0; j < n; j += UNROLL) {
        uint4 vr[UNROLL][CPL];
        // unguarded: past the wave's last slot, that slot's row is loaded again
#pragma unroll
        for (int uu = 0; uu < UNROLL; ++uu) {
          const uint4* vb =
              V + (int64_t)readlane_i32(ev, j + uu < n ? j + uu : n - 1) * row_chunks + cbase;
#pragma unroll
          for (int q = 0; q < CPL; ++q)
            vr[uu][q] = cvalid[q] ? vb[l + kWave * q] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int uu = 0; uu < UNROLL; ++uu) {
          if (j + uu < n) {
            const float wgt = readlane_f32(av, j + uu);
#pragma unroll
            for (int q = 0; q < CPL; ++q) {
              const uint4 c = vr[uu][q];
              if constexpr (BF16) {
                acc[q][0] = fmaf(wgt, bf16_lo(c.x), acc[q][0]);
                acc[q][1] = fmaf(wgt, bf16_hi(c.x), acc[q][1]);
                acc[q][2] = fmaf(wgt, bf16_lo(c.y), acc[q][2]);
                acc[q][3] = fmaf(wgt, bf16_hi(c.y), acc[q][3]);
                acc[q][4] = fmaf(wgt, bf16_lo(c.z), acc[q][4]);
                acc[q][5] = fmaf(wgt, bf16_hi(c.z), acc[q][5]);
                acc[q][6] = fmaf(wgt, bf16_lo(c.w), acc[q][6]);
                acc[q][7] = fmaf(wgt, bf16_hi(c.w), acc[q][7]);
              } else {
                acc[q][0] = fmaf(wgt, __uint_as_float(c.x), acc[q][0]);
                acc[q][1] = fmaf(wgt, __uint_as_float(c.y), acc[q][1]);
                acc[q][2] = fmaf(wgt, __uint_as_float(c.z), acc[q][2]);
                acc[q][3] = fmaf(wgt, __uint_as_float(c.w), acc[q][3]);
              }
            }
          }
        }
      }
    }
    // Wave w's partial row in y order: chunk l + 64 q of the split at floats (l + 64 q) EPC.
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; k += 4)
        *(float4*)&part[w][(l + kWave * q) * EPC + k] =
            make_float4(acc[q][k], acc[q][k + 1], acc[q][k + 2], acc[q][k + 3]);
    __syncthreads();
    const int nc = a.nchunks - cbase < CPL * kWave ? a.nchunks - cbase : CPL * kWave;
    float* yt = a.y + t * a.d + (int64_t)cbase * EPC;
    for (int j = threadIdx.x; j < nc * EPC; j += 64 * W) {
      float r = part[0][j];
#pragma unroll
      for (int ww = 1; ww < W; ++ww) r += part[ww][j];
      yt[j] = r;
    }
    __syncthreads();
  }
}

// Contribution rows (the accumulate written the way the method's scatter-add reads, but with a
// deterministic reduction): expert-major, each wave walks its range of the schedule like
// expert_dot_kernel, loads an expert's v row once per run and writes the fp32 row a[p] * v_e
// into row p of a [M, d] buffer, p being the token-major slot; reduce_contrib_kernel then sums
// each token's H*K rows in slot order. v is read once per run instead of once per task, at the
// price of writing and reading back M * d * 4 bytes.
struct ContribArgs {
  DotArgs s;       // schedule walk: perm, idx, sorted keys, M, N, hk, range
  const void* v;
  float* c;        // [M, d] fp32 contribution rows
  float* y;        // [T, d] fp32 out
  int64_t T;
  int d;
  int vchunks;     // 16-byte chunks of a v row
  int splits;      // reduce: waves per token (column splits of whole 64-chunk rows)
};

template <int CPL, bool BF16>
__global__ __launch_bounds__(256) void scatter_contrib_kernel(ContribArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int G = CPL >= 8 ? 2 : 4;
  const DotArgs& sa = a.s;
  const int l = lane_id();
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t s = range_start(sa, wave * sa.range);
  const int64_t e = range_start(sa, (wave + 1) * sa.range);
  if (s >= e) return;
  const uint4* V = (const uint4*)a.v;
  const int64_t row_chunks = a.vchunks;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = (l + kWave * q) < a.vchunks;
  int prev = -1;  // expert whose v row sits in vr[G - 1]
  uint4 vr[G][CPL];
#pragma unroll
  for (int i = 0; i < G; ++i)
#pragma unroll
    for (int q = 0; q < CPL; ++q) vr[i][q] = make_uint4(0, 0, 0, 0);
  for (int64_t b = s; b < e; b += kWave) {
    const int64_t pos = b + l;
    const bool ok = pos < e;
    const int key = ok ? key_at(sa, pos) : -1;
    const int p = ok ? task_at(sa, pos) : 0;
    const float av = ok ? sa.a[p] : 0.0f;
    const int cnt = (int)((e - b) < kWave ? (e - b) : kWave);
    for (int j0 = 0; j0 < cnt; j0 += G) {
      int ej[G], pj[G];
      float wj[G];
#pragma unroll
      for (int i = 0; i < G; ++i) {
        const int jj = (j0 + i < cnt) ? j0 + i : cnt - 1;
        ej[i] = readlane_i32(key, jj);
        pj[i] = readlane_i32(p, jj);
        wj[i] = readlane_f32(av, jj);
      }
#pragma unroll
      for (int i = 0; i < G; ++i) {
        if (j0 + i < cnt) {
          const int before = (i == 0) ? prev : ej[i - 1];
          if (ej[i] == before) {
#pragma unroll
            for (int q = 0; q < CPL; ++q) vr[i][q] = vr[(i + G - 1) % G][q];
          } else {
            load_row<CPL>(vr[i], V + (int64_t)ej[i] * row_chunks, cv);
          }
        }
      }
#pragma unroll
      for (int i = 0; i < G; ++i) {
        if (j0 + i < cnt) {
          float4* row = (float4*)(a.c + (int64_t)pj[i] * a.d);
#pragma unroll
          for (int q = 0; q < CPL; ++q) {
            if (!cv[q]) continue;
            const uint4 c = vr[i][q];
            const int o = (l + kWave * q) * (EPC / 4);
            const float w = wj[i];
            if constexpr (BF16) {
              row[o] = make_float4(w * bf16_lo(c.x), w * bf16_hi(c.x), w * bf16_lo(c.y),
                                   w * bf16_hi(c.y));
              row[o + 1] = make_float4(w * bf16_lo(c.z), w * bf16_hi(c.z), w * bf16_lo(c.w),
                                       w * bf16_hi(c.w));
            } else {
              row[o] = make_float4(w * __uint_as_float(c.x), w * __uint_as_float(c.y),
                                   w * __uint_as_float(c.z), w * __uint_as_float(c.w));
            }
          }
        }
      }
      const int last = (cnt - j0 < G ? cnt - j0 : G) - 1;
#pragma unroll
      for (int i = 0; i < G - 1; ++i)
        if (i == last) {
#pragma unroll
          for (int q = 0; q < CPL; ++q) vr[G - 1][q] = vr[i][q];
        }
      prev = ej[last];
    }
  }
}

// y_t = sum over t's slots s (in order) of row t*H*K + s of the contribution buffer, fp32.
// One wave per (token, column split); lane l holds float4 columns l + 64 q of the split.
template <int CPL>
__global__ __launch_bounds__(256) void reduce_contrib_kernel(ContribArgs a) {
  constexpr int UNROLL = CPL >= 16 ? 2 : 4;
  const int l = lane_id();
  const int f4 = a.d / 4;  // float4 columns per row
  const int hk = a.s.hk;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t wt = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); wt < a.T * a.splits;
       wt += stride) {
    const int64_t t = wt / a.splits;
    const int cbase = (int)(wt % a.splits) * CPL * kWave;
    bool cvalid[CPL];
#pragma unroll
    for (int q = 0; q < CPL; ++q) cvalid[q] = (cbase + l + kWave * q) < f4;
    float4 acc[CPL];
#pragma unroll
    for (int q = 0; q < CPL; ++q) acc[q] = make_float4(0.f, 0.f, 0.f, 0.f);
    const float4* base = (const float4*)(a.c + t * hk * (int64_t)a.d) + cbase + l;
    for (int s0 = 0; s0 < hk; s0 += UNROLL) {
      float4 r[UNROLL][CPL];
#pragma unroll
      for (int u = 0; u < UNROLL; ++u)
#pragma unroll
        for (int q = 0; q < CPL; ++q)
          r[u][q] = (s0 + u < hk && cvalid[q]) ? base[(int64_t)(s0 + u) * f4 + kWave * q]
                                               : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        if (s0 + u < hk) {
#pragma unroll
          for (int q = 0; q < CPL; ++q) {
            acc[q].x += r[u][q].x;
            acc[q].y += r[u][q].y;
            acc[q].z += r[u][q].z;
            acc[q].w += r[u][q].w;
          }
        }
      }
    }
    float4* yt = (float4*)(a.y + t * a.d) + cbase + l;
#pragma unroll
    for (int q = 0; q < CPL; ++q)
      if (cvalid[q]) yt[kWave * q] = acc[q];
  }
}

// Token-centric execution (the scheduling ablation): one wavefront per token keeps x_t in
// registers and, G slots at a time in (head, k) order, gathers each slot's u and v rows
// together, forms a = g * act(x_t . u_e) exactly as expert_dot_kernel does and adds a * v_e
// into the fp32 row as accumulate_kernel does. Same operations in the same order, so y equals
// the scheduled path's bit for bit; every u row is read once per task instead of once per run.
struct TokenArgs {
  const void* x;
  const void* u;
  const void* v;
  const int32_t* idx;
  const float* gates;
  float* y;
  int64_t T;
  int64_t N;
  int d;
  int hk;
  int act;
  int nchunks;
};

template <int CPL, bool BF16>
__global__ __launch_bounds__(256) void token_centric_kernel(TokenArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int G = CPL >= 16 ? 1 : (CPL >= 8 ? 2 : 4);
  const int l = lane_id();
  const uint4* X = (const uint4*)a.x;
  const uint4* U = (const uint4*)a.u;
  const uint4* V = (const uint4*)a.v;
  const int64_t row_chunks = a.nchunks;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = (l + kWave * q) < a.nchunks;
  const int64_t stride = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < a.T; t += stride) {
    uint4 xr[CPL];
    load_row<CPL>(xr, X + t * row_chunks, cv);
    float acc[CPL][EPC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[q][k] = 0.0f;
    for (int sb = 0; sb < a.hk; sb += kWave) {
      const int sl = sb + l;
      const bool valid = sl < a.hk;
      const int ev = valid ? clamp_i(a.idx[t * a.hk + sl], a.N) : 0;
      const float gv = valid ? a.gates[t * a.hk + sl] : 0.0f;
      const int n = a.hk - sb < kWave ? a.hk - sb : kWave;
      for (int j = 0; j < n; j += G) {
        uint4 ur[G][CPL], vr[G][CPL];
        float gj[G];
#pragma unroll
        for (int i = 0; i < G; ++i) {
          const int jj = j + i < n ? j + i : n - 1;
          const int e = readlane_i32(ev, jj);
          gj[i] = readlane_f32(gv, jj);
          load_row<CPL>(ur[i], U + (int64_t)e * row_chunks, cv);
          load_row<CPL>(vr[i], V + (int64_t)e * row_chunks, cv);
        }
#pragma unroll
        for (int i = 0; i < G; ++i) {
          if (j + i < n) {
            float h = 0.0f;
#pragma unroll
            for (int q = 0; q < CPL; ++q) h = chunk_dot<BF16>(ur[i][q], xr[q], h);
            const float w = gj[i] * activation(a.act, wave_sum_uniform(h));
#pragma unroll
            for (int q = 0; q < CPL; ++q) {
              const uint4 c = vr[i][q];
              if constexpr (BF16) {
                acc[q][0] = fmaf(w, bf16_lo(c.x), acc[q][0]);
                acc[q][1] = fmaf(w, bf16_hi(c.x), acc[q][1]);
                acc[q][2] = fmaf(w, bf16_lo(c.y), acc[q][2]);
                acc[q][3] = fmaf(w, bf16_hi(c.y), acc[q][3]);
                acc[q][4] = fmaf(w, bf16_lo(c.z), acc[q][4]);
                acc[q][5] = fmaf(w, bf16_hi(c.z), acc[q][5]);
                acc[q][6] = fmaf(w, bf16_lo(c.w), acc[q][6]);
                acc[q][7] = fmaf(w, bf16_hi(c.w), acc[q][7]);
              } else {
                acc[q][0] = fmaf(w, __uint_as_float(c.x), acc[q][0]);
                acc[q][1] = fmaf(w, __uint_as_float(c.y), acc[q][1]);
                acc[q][2] = fmaf(w, __uint_as_float(c.z), acc[q][2]);
                acc[q][3] = fmaf(w, __uint_as_float(c.w), acc[q][3]);
              }
            }
          }
        }
      }
    }
    float4* yt = (float4*)(a.y + t * a.d);
#pragma unroll
    for (int q = 0; q < CPL; ++q) {
      if (!cv[q]) continue;
      const int c = l + kWave * q;
#pragma unroll
      for (int k = 0; k < EPC; k += 4)
        yt[(c * EPC + k) / 4] = make_float4(acc[q][k], acc[q][k + 1], acc[q][k + 2], acc[q][k + 3]);
    }
  }
}

template <bool BF16>
hipError_t dispatch_token(int cpl, dim3 grid, hipStream_t st, const TokenArgs& a) {
  switch (cpl) {
    case 1: hipLaunchKernelGGL((token_centric_kernel<1, BF16>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((token_centric_kernel<2, BF16>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((token_centric_kernel<4, BF16>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((token_centric_kernel<8, BF16>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((token_centric_kernel<16, BF16>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

template <bool BF16>
hipError_t dispatch_dot(int cpl, dim3 grid, hipStream_t st, const DotArgs& a) {
  const bool full = a.nchunks == cpl * kWave;
#define OMNIMOE_DOT(C_)                                                                    \
  do {                                                                                     \
    if (full) hipLaunchKernelGGL((expert_dot_kernel<C_, BF16, true>), grid, dim3(256), 0, st, a); \
    else hipLaunchKernelGGL((expert_dot_kernel<C_, BF16, false>), grid, dim3(256), 0, st, a);    \
  } while (0)
  switch (cpl) {
    case 1: OMNIMOE_DOT(1); break;
    case 2: OMNIMOE_DOT(2); break;
    case 4: OMNIMOE_DOT(4); break;
    case 8: OMNIMOE_DOT(8); break;
    default: OMNIMOE_DOT(16); break;
  }
#undef OMNIMOE_DOT
  return hipGetLastError();
}

// ---------------------------------------------------------------- slot order (no schedule)
// Where the expert-major order saves no memory traffic, the layer runs the dot in slot order
// without a schedule: wave v takes slots 2v and 2v + 1, reads their experts and gates and loads
// both u rows and token rows at once. That is the case (measured: bench, layer per call)
//   - for a decode step (M <= 8192): 64 tokens pick ~8165 distinct experts of 2^20 in 8192
//     slots, so there is no u row to share;
//   - when tasks are at most half the experts (M <= N / 2, about 1.1 tasks per active expert
//     under uniform routing): 2048 tokens on the 2^20-expert tables, 0.611 -> 0.505 ms;
//   - when the u table fits in half the 256 MB MALL, where a re-read costs no HBM traffic: 4096
//     tokens on 2^16 experts of d = 512, 0.201 -> 0.148 ms.
// With 2.3 tasks per active expert and 4 GiB tables (16384 tokens on 2^20 experts) the schedule
// pays: 3.54 against 3.64 ms. Each a[p] is summed exactly as expert_dot_kernel sums it, so the
// two kernels give identical a.
constexpr int kSlotDotMaxTasks = 8192;
constexpr int64_t kSlotDotMaxTableBytes = 128ll << 20;

template <int CPL, bool BF16, bool FULL>
__global__ __launch_bounds__(256) void slot_dot_kernel(DotArgs a) {
  constexpr int G = CPL >= 8 ? 1 : 2;  // slots per wave, all in flight
  const int l = lane_id();
  const int64_t p0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * G;
  const uint4* X = (const uint4*)a.x;
  const uint4* U = (const uint4*)a.u;
  bool cv[CPL];
#pragma unroll
  for (int q = 0; q < CPL; ++q) cv[q] = FULL || (l + kWave * q) < a.nchunks;
  uint4 ur[G][CPL], xr[G][CPL];
  float gj[G];
  int ej[G];
  // Every slot's expert and gate first, then the token rows (they need no index), then the u
  // rows: loads complete in order, so an index load issued behind rows would make the u row
  // that needs it wait for those rows as well. The loads are unconditional (a slot past the
  // end reads the last slot again and is not stored) so that the compiler can count them.
  int64_t pj[G];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    pj[i] = p0 + i < a.M ? p0 + i : a.M - 1;
    ej[i] = a.idx[pj[i]];
    gj[i] = a.gates[pj[i]];
  }
#pragma unroll
  for (int i = 0; i < G; ++i) load_row<CPL>(xr[i], X + (pj[i] / a.hk) * a.nchunks, cv);
#pragma unroll
  for (int i = 0; i < G; ++i)
    load_row_nt<CPL>(ur[i], U + (int64_t)clamp_i(ej[i], a.N) * a.nchunks, cv);
  // lane i finishes slot p0 + i: one activation for the wave's slots (the sums are formed for
  // every slot, so that no load is moved into a branch behind another slot's work)
  float hv = 0.0f, gv = 0.0f;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    float acc = 0.0f;
#pragma unroll
    for (int q = 0; q < CPL; ++q) acc = chunk_dot<BF16>(ur[i][q], xr[i][q], acc);
    const float hs = wave_sum_uniform(acc);
    if (l == i) {
      hv = hs;
      gv = gj[i];
    }
  }
  if (l < G && p0 + l < a.M) a.a[p0 + l] = gv * activation(a.act, hv);
}

template <bool BF16>
hipError_t dispatch_slot_dot(int cpl, dim3 grid, hipStream_t st, const DotArgs& a) {
  const bool full = a.nchunks == cpl * kWave;
#define OMNIMOE_SLOT(C_)                                                                    \
  do {                                                                                      \
    if (full) hipLaunchKernelGGL((slot_dot_kernel<C_, BF16, true>), grid, dim3(256), 0, st, a); \
    else hipLaunchKernelGGL((slot_dot_kernel<C_, BF16, false>), grid, dim3(256), 0, st, a);    \
  } while (0)
  switch (cpl) {
    case 1: OMNIMOE_SLOT(1); break;
    case 2: OMNIMOE_SLOT(2); break;
    case 4: OMNIMOE_SLOT(4); break;
    case 8: OMNIMOE_SLOT(8); break;
    default: OMNIMOE_SLOT(16); break;
  }
#undef OMNIMOE_SLOT
  return hipGetLastError();
}

// Sixteen waves per workgroup when a wave holds at most two chunks of a row (registers for
// eight rows in flight, at most 64 KiB of partial rows in LDS) and each wave still gets a few
// slots; four otherwise.
// FULL when each wave's column split is exactly CPL * 64 chunks of the row.
template <bool BF16>
hipError_t dispatch_acc_slots(int cpl, int hk, dim3 grid, hipStream_t st, const AccArgs& a) {
  const bool full = a.nchunks == a.splits * cpl * kWave;
#define OMNIMOE_ACCS(W_, C_)                                                                    \
  do {                                                                                          \
    if (full) hipLaunchKernelGGL((accumulate_slots_kernel<W_, C_, BF16, true>), grid, dim3(64 * W_), 0, st, a); \
    else hipLaunchKernelGGL((accumulate_slots_kernel<W_, C_, BF16, false>), grid, dim3(64 * W_), 0, st, a);     \
  } while (0)
  if (cpl <= 2 && hk >= 64) {
    if (cpl == 1) OMNIMOE_ACCS(16, 1);
    else OMNIMOE_ACCS(16, 2);
    return hipGetLastError();
  }
  switch (cpl) {
    case 1: OMNIMOE_ACCS(4, 1); break;
    case 2: OMNIMOE_ACCS(4, 2); break;
    case 4: OMNIMOE_ACCS(4, 4); break;
    case 8: OMNIMOE_ACCS(4, 8); break;
    default: OMNIMOE_ACCS(4, 16); break;
  }
#undef OMNIMOE_ACCS
  return hipGetLastError();
}

template <bool BF16>
hipError_t dispatch_acc(int cpl, dim3 grid, hipStream_t st, const AccArgs& a) {
  switch (cpl) {
    case 1: hipLaunchKernelGGL((accumulate_kernel<1, BF16>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((accumulate_kernel<2, BF16>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((accumulate_kernel<4, BF16>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((accumulate_kernel<8, BF16>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((accumulate_kernel<16, BF16>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

template <bool BF16>
hipError_t dispatch_scatter(int cpl, dim3 grid, hipStream_t st, const ContribArgs& a) {
  switch (cpl) {
    case 1: hipLaunchKernelGGL((scatter_contrib_kernel<1, BF16>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((scatter_contrib_kernel<2, BF16>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((scatter_contrib_kernel<4, BF16>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((scatter_contrib_kernel<8, BF16>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((scatter_contrib_kernel<16, BF16>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

hipError_t dispatch_reduce_contrib(int cpl, dim3 grid, hipStream_t st, const ContribArgs& a) {
  switch (cpl) {
    case 1: hipLaunchKernelGGL((reduce_contrib_kernel<1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((reduce_contrib_kernel<2>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((reduce_contrib_kernel<4>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((reduce_contrib_kernel<8>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((reduce_contrib_kernel<16>), grid, dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

// Chunks per lane, rounded up to a power of two.
int chunks_per_lane(int nchunks) {
  int c = 1;
  while (c * kWave < nchunks) c <<= 1;
  return c;
}

}  // namespace

hipError_t launch_expert_dot(const Shape& s, const void* x, const void* u, const int32_t* idx,
                             const float* gates, const int32_t* perm, const int32_t* sorted_keys,
                             float* abuf, hipStream_t st) {
  if (s.M == 0) return hipSuccess;
  DotArgs a;
  a.x = x;
  a.u = u;
  a.idx = idx;
  a.gates = gates;
  a.perm = perm;
  a.sk = sorted_keys;
  a.a = abuf;
  a.M = s.M;
  a.N = s.N;
  a.d = s.d;
  a.hk = s.hk;
  a.act = s.act;
  a.nchunks = s.bf16 ? s.d / 8 : s.d / 4;
  // 8 tasks per wave when experts average at most 4 tasks, 16 below 8 (fewer tasks in flight per
  // XCD keeps its stretch of token rows in L2), 64 otherwise (a range starts inside an expert's run
  // only when the run is longer than the range, and each such start reads u again); fewer, down
  // to one, so that small batches still give at least 2048 waves.
  a.range = s.M <= 4 * s.N ? 8 : (s.M < 8 * s.N ? 16 : 64);
  while (a.range > 1 && s.M < (int64_t)a.range * 2048) a.range >>= 1;
  const int64_t waves = (s.M + a.range - 1) / a.range;
  dim3 grid((unsigned)((waves + 3) / 4));
  const int cpl = chunks_per_lane(a.nchunks);
  return s.bf16 ? dispatch_dot<true>(cpl, grid, st, a) : dispatch_dot<false>(cpl, grid, st, a);
}

bool slot_dot(const Shape& s) {
  const int64_t table = s.N * (int64_t)s.d * (s.bf16 ? 2 : 4);
  return s.M > 0 &&
         (s.M <= kSlotDotMaxTasks || 2 * s.M <= s.N || table <= kSlotDotMaxTableBytes);
}

hipError_t launch_slot_dot(const Shape& s, const void* x, const void* u, const int32_t* idx,
                           const float* gates, float* abuf, hipStream_t st) {
  if (s.M == 0) return hipSuccess;
  DotArgs a;
  a.x = x;
  a.u = u;
  a.idx = idx;
  a.gates = gates;
  a.perm = nullptr;
  a.sk = nullptr;
  a.a = abuf;
  a.M = s.M;
  a.N = s.N;
  a.d = s.d;
  a.hk = s.hk;
  a.act = s.act;
  a.nchunks = s.bf16 ? s.d / 8 : s.d / 4;
  a.range = 1;
  const int cpl = chunks_per_lane(a.nchunks);
  const int64_t per_wave = cpl >= 8 ? 1 : 2;
  const int64_t waves = (s.M + per_wave - 1) / per_wave;
  const dim3 grid((unsigned)((waves + 3) / 4));
  return s.bf16 ? dispatch_slot_dot<true>(cpl, grid, st, a)
                : dispatch_slot_dot<false>(cpl, grid, st, a);
}

hipError_t launch_accumulate(const Shape& s, const void* v, const int32_t* idx, const float* abuf,
                             float* y, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  AccArgs a;
  a.v = v;
  a.idx = idx;
  a.a = abuf;
  a.y = y;
  a.T = s.T;
  a.N = s.N;
  a.d = s.d;
  a.hk = s.hk;
  a.nchunks = s.bf16 ? s.d / 8 : s.d / 4;
  // Few tokens: split each token's row over several waves (whole 64-chunk rows each).
  const int rows64 = (a.nchunks + kWave - 1) / kWave;
  int splits = 1;
  while (splits < rows64 && s.T * splits < 1024 && rows64 % (splits * 2) == 0) splits *= 2;
  a.splits = splits;
  const int cpl = chunks_per_lane((a.nchunks + splits - 1) / splits);
  if (s.T * splits < 1024 && s.hk >= 16) {
    // still few waves: a workgroup per (token, column split), slots shared by its waves
    const int64_t units = s.T * splits;
    const dim3 grid((unsigned)(units < 16384 ? units : 16384));
    return s.bf16 ? dispatch_acc_slots<true>(cpl, s.hk, grid, st, a)
                  : dispatch_acc_slots<false>(cpl, s.hk, grid, st, a);
  }
  int64_t blocks = (s.T * splits + 3) / 4;
  if (blocks > 16384) blocks = 16384;
  return s.bf16 ? dispatch_acc<true>(cpl, dim3((unsigned)blocks), st, a)
                : dispatch_acc<false>(cpl, dim3((unsigned)blocks), st, a);
}

hipError_t launch_token_centric(const Shape& s, const void* x, const void* u, const void* v,
                                const int32_t* idx, const float* gates, float* y,
                                hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  TokenArgs a;
  a.x = x;
  a.u = u;
  a.v = v;
  a.idx = idx;
  a.gates = gates;
  a.y = y;
  a.T = s.T;
  a.N = s.N;
  a.d = s.d;
  a.hk = s.hk;
  a.act = s.act;
  a.nchunks = s.bf16 ? s.d / 8 : s.d / 4;
  int64_t blocks = (s.T + 3) / 4;
  if (blocks > 16384) blocks = 16384;
  const int cpl = chunks_per_lane(a.nchunks);
  return s.bf16 ? dispatch_token<true>(cpl, dim3((unsigned)blocks), st, a)
                : dispatch_token<false>(cpl, dim3((unsigned)blocks), st, a);
}

hipError_t launch_expert_contrib(const Shape& s, const void* x, const void* u, const void* v,
                                 const int32_t* idx, const float* gates, const int32_t* perm,
                                 float* abuf, float* cbuf, float* y, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  hipError_t e = launch_expert_dot(s, x, u, idx, gates, perm, nullptr, abuf, st);
  if (e != hipSuccess || s.M == 0) return e;
  ContribArgs a;
  a.s.x = x;
  a.s.u = u;
  a.s.idx = idx;
  a.s.gates = gates;
  a.s.perm = perm;
  a.s.sk = nullptr;
  a.s.a = abuf;
  a.s.M = s.M;
  a.s.N = s.N;
  a.s.d = s.d;
  a.s.hk = s.hk;
  a.s.act = s.act;
  a.s.nchunks = s.bf16 ? s.d / 8 : s.d / 4;
  a.s.range = 64;
  while (a.s.range > 1 && s.M < (int64_t)a.s.range * 2048) a.s.range >>= 1;
  a.v = v;
  a.c = cbuf;
  a.y = y;
  a.T = s.T;
  a.d = s.d;
  a.vchunks = a.s.nchunks;
  const int64_t waves = (s.M + a.s.range - 1) / a.s.range;
  const dim3 grid((unsigned)((waves + 3) / 4));
  const int cpl = chunks_per_lane(a.vchunks);
  e = s.bf16 ? dispatch_scatter<true>(cpl, grid, st, a) : dispatch_scatter<false>(cpl, grid, st, a);
  if (e != hipSuccess) return e;
  // Reduce: float4 columns, split over waves while there are few tokens.
  const int f4 = s.d / 4;
  const int rows64 = (f4 + kWave - 1) / kWave;
  int splits = 1;
  while ((f4 + splits - 1) / splits > 16 * kWave) splits *= 2;  // at most 16 float4 per lane
  while (splits < rows64 && s.T * splits < 1024 && rows64 % (splits * 2) == 0) splits *= 2;
  a.splits = splits;
  int64_t blocks = (s.T * splits + 3) / 4;
  if (blocks > 16384) blocks = 16384;
  return dispatch_reduce_contrib(chunks_per_lane((f4 + splits - 1) / splits),
                                 dim3((unsigned)blocks), st, a);
}

}  // namespace omnimoe
