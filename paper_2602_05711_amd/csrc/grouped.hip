// Grouped expert GEMM of Eq. 14 for a schedule with groups of B > 1 active experts: the
// activations G_q (.) act(X_q W_q^T) of group q are formed as dense tiles on MFMA, X_q being
// the group's distinct tokens (its slots) and W_q the u rows of its experts. Only the entries
// that are tasks are kept: a[p] = g_p * act(x_t . u_e) for every task p of the group.
//
// Work tile: 256 slots x 32 NJ experts of one group per workgroup of four waves (each wave 64
// slots x 32 NJ experts, 2 NJ accumulators of v_mfma_f32_32x32x16_bf16); NJ = 2 (64 experts)
// for groups of up to 64, else 5 (160 experts), so that one load of a token row serves more
// experts. k steps of 64 go through two LDS stages filled straight from global memory with
// global_load_lds_dwordx4: every lane supplies its own row address, so the token rows (x at the
// slots' tokens) and the expert rows (u at the group's experts) are gathered on the way into
// LDS. LDS rows are 128 B; chunk j of row r sits at position j ^ ((r >> 1) & 7), so the 16 rows
// read by one operand load fall in distinct banks. bf16 products are exact and accumulate in
// fp32, as in the per-task kernel.
//
// Epilogue: the fp32 tile goes to LDS (over the stages; in two halves of 128 slot rows when it
// does not fit at once) with the tile's slot offsets, and the workgroup walks the tasks of those
// slots (one contiguous run of sorted positions) 256 at a time; those whose expert lies in the
// tile (its place in the group, from the schedule's packed key) find their slot row by binary
// search in the offsets, read their entry and write a[p].
//
// Tiles are numbered group by group (slot tiles major, expert tiles fastest), so consecutive
// tiles share their token rows and the group's u rows stay in the XCD's L2; each XCD takes one
// contiguous range of tiles and each workgroup a contiguous run inside it, so the group search
// is done once per workgroup and then advances. With groups of up to 64 experts and six or more
// slot tiles per group on average the XCDs split the tiles by token range instead (below).
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int kThreads = 256;
constexpr int kK = 64;      // k per stage
constexpr int kRow = kK * 2;  // bytes per LDS row
static_assert(kGroupSlots == 4 * 64, "four waves of 64 slot rows");

template <int NJ>
struct TileShape {
  static constexpr int kExperts = 32 * NJ;
  static constexpr int kStage = (kGroupSlots + kExperts) * kRow;
  static constexpr int kHStride = kExperts + 1;  // floats per epilogue row
  // slot rows per epilogue pass: all 256 if the tile and the offsets fit in the two stages
  static constexpr int kRowsPerPass =
      kGroupSlots * kHStride * 4 + (kGroupSlots + 1) * 4 <= 2 * kStage ? kGroupSlots
                                                                        : kGroupSlots / 2;
  static constexpr int kOffBase = kRowsPerPass * kHStride * 4;
  static_assert(kOffBase + (kGroupSlots + 1) * 4 <= 2 * kStage, "the epilogue fits the stages");
};

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

struct GroupedDotArgs {
  const uint16_t* x;
  const uint16_t* u;
  const float* gates;
  const int32_t* perm;
  const int32_t* active;
  const int32_t* n_active;
  const int32_t* key;
  const int32_t* slot_token;
  const int32_t* slot_off;
  const int32_t* grp_slot;
  const int32_t* grp_tile;
  const int32_t* counters;
  float* a;
  int64_t M, N, G;
  int d, B, act, gbits;
};

__device__ __forceinline__ int32_t clamp_i32(int32_t v, int64_t n) {
  return v < 0 ? 0 : (v >= n ? (int32_t)(n - 1) : v);
}

template <int NJ>
__global__ __launch_bounds__(kThreads, 1) void grouped_dot_kernel(GroupedDotArgs a) {
  using TS = TileShape<NJ>;
  constexpr int TE = TS::kExperts;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  const int n_act = *a.n_active;
  int64_t ng = ((int64_t)n_act + a.B - 1) / a.B;
  if (ng > a.G) ng = a.G;
  const int total = a.counters[1];
  if (ng <= 0 || total <= 0) return;
  // each XCD a contiguous range of tiles, each workgroup a contiguous run inside it
  constexpr int kXcds = 8;
  const int xcd = blockIdx.x % kXcds;
  const int blocks_per_xcd = gridDim.x / kXcds;
  const int per_xcd = (total + kXcds - 1) / kXcds;
  const int x_lo = xcd * per_xcd;
  const int x_hi = min(total, x_lo + per_xcd);
  const int per_block = (per_xcd + blocks_per_xcd - 1) / blocks_per_xcd;
  const int t_lo = x_lo + (blockIdx.x / kXcds) * per_block;
  const int t_hi = min(x_hi, t_lo + per_block);
  // group of the first tile (contiguous mapping): the last q < ng with grp_tile[q] <= t_lo
  int q = 0;
  if (t_lo < t_hi) {
    int lo = 0, hi = (int)ng - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.grp_tile[mid] <= t_lo) lo = mid; else hi = mid - 1;
    }
    q = lo;
  }
  const int frow = l & 31;
  const int fk = l >> 5;  // 16-byte chunk within a 16-wide k step
  const int sw = swz(frow);
  const int KT = a.d / kK;
  // One work tile: slot tile stl and expert tile et of group q (the same on every lane).
  auto run_tile = [&](int q, int stl, int et) {
    const int s_q = a.grp_slot[q];
    const int tq = a.grp_slot[q + 1] - s_q;
    const int e_q = q * a.B;
    const int bq = min(a.B, n_act - e_q);
    const int s0 = s_q + stl * kGroupSlots;
    const int ns = min(kGroupSlots, tq - stl * kGroupSlots);
    const int r0 = e_q + et * TE;
    const int ne = min(TE, bq - et * TE);
    // Loader: instruction i of wave w fills 8 LDS rows; lane l writes position l % 8 of row
    // l / 8 of them, i.e. global chunk (l % 8) ^ swz(row). Rows past the tile's slots or
    // experts load the tile's first row (never read back).
    const uint16_t* ga[8];
    const uint16_t* gb[NJ];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = (w * 8 + i) * 8 + (l >> 3);
      const int j = (l & 7) ^ swz(r);
      const int32_t tok = a.slot_token[s0 + (r < ns ? r : 0)];
      ga[i] = a.x + (int64_t)tok * a.d + j * 8;
    }
#pragma unroll
    for (int i = 0; i < NJ; ++i) {
      const int r = (w * NJ + i) * 8 + (l >> 3);
      const int j = (l & 7) ^ swz(r);
      const int32_t e = clamp_i32(a.active[r0 + (r < ne ? r : 0)], a.N);
      gb[i] = a.u + (int64_t)e * a.d + j * 8;
    }
    auto issue = [&](int stage, int k0) {
      unsigned char* base = smem + stage * TS::kStage;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_global_load_lds((const void*)(ga[i] + k0),
                                         (lds_ptr_t)(base + (w * 8 + i) * 8 * kRow), 16, 0, 0);
#pragma unroll
      for (int i = 0; i < NJ; ++i)
        __builtin_amdgcn_global_load_lds(
            (const void*)(gb[i] + k0),
            (lds_ptr_t)(base + kGroupSlots * kRow + (w * NJ + i) * 8 * kRow), 16, 0, 0);
    };
    int a_off[2], b_off[NJ];  // LDS row offsets of this lane's operand rows
#pragma unroll
    for (int i = 0; i < 2; ++i) a_off[i] = (w * 64 + i * 32 + frow) * kRow;
#pragma unroll
    for (int j = 0; j < NJ; ++j) b_off[j] = kGroupSlots * kRow + (j * 32 + frow) * kRow;
    auto frag = [&](const unsigned char* st, int off, int ks) -> bf16x8 {
      return *(const bf16x8*)(st + off + (((ks * 2 + fk) ^ sw) << 4));
    };
    f32x16 acc[2][NJ];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    issue(0, 0);
    wait_vm0();
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < KT) issue(cur ^ 1, (kt + 1) * kK);
      const unsigned char* st = smem + cur * TS::kStage;
      bf16x8 fa[2][2], fb[2][NJ];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[0][i] = frag(st, a_off[i], 0);
#pragma unroll
      for (int j = 0; j < NJ; ++j) fb[0][j] = frag(st, b_off[j], 0);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int c = ks & 1;
        if (ks + 1 < 4) {
#pragma unroll
          for (int i = 0; i < 2; ++i) fa[c ^ 1][i] = frag(st, a_off[i], ks + 1);
#pragma unroll
          for (int j = 0; j < NJ; ++j) fb[c ^ 1][j] = frag(st, b_off[j], ks + 1);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[c][i], fb[c][j], acc[i][j],
                                                                0, 0, 0);
      }
      wait_vm0();
      __syncthreads();
    }
    // accumulator element r of block (i, j) of wave w: slot row 64 w + 32 i + 8 (r / 4) +
    // 4 (l / 32) + r % 4, expert column 32 j + l % 32
    float* H = (float*)smem;
    int32_t* offs = (int32_t*)(smem + TS::kOffBase);  // offs[r] = first position of slot s0 + r
    for (int r = tid; r <= ns; r += kThreads) offs[r] = a.slot_off[s0 + r];
    const int c0 = et * TE;
#pragma unroll
    for (int pass = 0; pass < kGroupSlots / TS::kRowsPerPass; ++pass) {
      const int row0 = pass * TS::kRowsPerPass;  // first slot row held in H this pass
      if (w * 64 >= row0 && w * 64 < row0 + TS::kRowsPerPass) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              H[(w * 64 - row0 + i * 32 + (r >> 2) * 8 + (l >> 5) * 4 + (r & 3)) * TS::kHStride +
                j * 32 + (l & 31)] = acc[i][j][r];
      }
      __syncthreads();
      const int r_hi = min(ns, row0 + TS::kRowsPerPass);
      if (row0 < r_hi) {
        const int p_lo = offs[row0], p_hi = offs[r_hi];
        for (int pos = p_lo + tid; pos < p_hi; pos += kThreads) {
          const int c = (int)((uint32_t)a.key[pos] >> a.gbits) - c0;
          if (c >= 0 && c < ne) {
            int lo = row0, hi = r_hi - 1;  // the last slot r with offs[r] <= pos
            while (lo < hi) {
              const int mid = (lo + hi + 1) >> 1;
              if (offs[mid] <= pos) lo = mid; else hi = mid - 1;
            }
            const int32_t p = clamp_i32(a.perm[pos], a.M);
            a.a[p] = a.gates[p] * activation(a.act, H[(lo - row0) * TS::kHStride + c]);
          }
        }
      }
      __syncthreads();
    }
  };

  if (NJ == 2 && total >= 6 * ng) {
    // Groups of up to 64 experts with many slot tiles each: a group's slots are in token order,
    // so its slot tiles cover successive eighths of the tokens. XCD x takes the slot tiles stl
    // with (8 stl + 4) / n_st = x of every group (n_st slot tiles), about an eighth of the
    // tokens, whose rows then stay in its L2 across groups; workgroup r of the XCD takes every
    // R-th of those tiles in group order. Every wave computes the same tile sequence from the
    // same data. (Each XCD now reads every group's u rows; with the small groups that costs
    // less than the token rows saved, with 160-expert tiles it does not, measured.)
    const int r = blockIdx.x / kXcds, R = blocks_per_xcd;
    int seen = 0;  // tiles of this XCD in the groups before this batch
    for (int qb = 0; qb < (int)ng; qb += kWave) {
      const int qq = qb + l;
      int cnt = 0, lo_st = 0, n_et = 1;
      if (qq < ng) {
        const int n_st = (a.grp_slot[qq + 1] - a.grp_slot[qq] + kGroupSlots - 1) / kGroupSlots;
        n_et = (min(a.B, n_act - qq * a.B) + TE - 1) / TE;
        const int lo8 = xcd * n_st - 4, hi8 = (xcd + 1) * n_st - 4;
        lo_st = lo8 <= 0 ? 0 : (lo8 + 7) / 8;
        const int hi_st = hi8 <= 0 ? 0 : min(n_st, (hi8 + 7) / 8);
        cnt = hi_st > lo_st ? (hi_st - lo_st) * n_et : 0;
      }
      const int ex = wave_excl_scan_i32(cnt);
      const int first = seen + ex;  // XCD-stream index of this lane's first tile
      const int skip = ((r - first) % R + R) % R;
      uint64_t mine = __ballot(skip < cnt);
      while (mine) {
        const int L = __ffsll((unsigned long long)mine) - 1;
        mine &= mine - 1;
        const int cL = readlane_i32(cnt, L), lL = readlane_i32(lo_st, L);
        const int eL = readlane_i32(n_et, L), sL = readlane_i32(skip, L);
        for (int i = sL; i < cL; i += R) run_tile(qb + L, lL + i / eL, i % eL);
      }
      seen += readlane_i32(ex + cnt, kWave - 1);
    }
    return;
  }
  for (int tile = t_lo; tile < t_hi; ++tile) {
    while (q + 1 < ng && a.grp_tile[q + 1] <= tile) ++q;
    const int bq = min(a.B, n_act - q * a.B);
    const int n_et = (bq + TE - 1) / TE;
    const int local = tile - a.grp_tile[q];
    const int stl = local / n_et;
    run_tile(q, stl, local - stl * n_et);
  }
}

// ---------------------------------------------------------------- second product per group
// O[s] = sum over the tasks of slot s (sorted positions slot_off[s] .. slot_off[s + 1], one
// token's tasks in one group) of a_p v_e, in position order, fp32. One wave per slot; each
// XCD takes a contiguous range of slots (workgroup b runs on XCD b % 8), i.e. whole groups one
// after the other, so a group's v rows are fetched from HBM once and then found in that XCD's
// L2. Columns go in chunks of 512 (eight per lane, one 16-byte load of bf16 per task).
struct GroupRowsArgs {
  const uint16_t* v;
  const int32_t* idx;
  const int32_t* perm;
  const float* a;
  const int32_t* slot_off;
  const int32_t* counters;
  float* rows;
  int64_t M, N, n_max;
  int d;
};

__device__ __forceinline__ void fma_bf16x8(float (&acc)[8], float w, uint4 q) {
  acc[0] += w * bf16_lo(q.x); acc[1] += w * bf16_hi(q.x);
  acc[2] += w * bf16_lo(q.y); acc[3] += w * bf16_hi(q.y);
  acc[4] += w * bf16_lo(q.z); acc[5] += w * bf16_hi(q.z);
  acc[6] += w * bf16_lo(q.w); acc[7] += w * bf16_hi(q.w);
}

// Columns in passes of 512 CH (CH 16-byte bf16 loads per lane and task, 8 CH fp32 sums per
// lane); the tasks of a slot four at a time, their rows all requested before the sums.
template <int CH>
__device__ __forceinline__ void group_row_pass(const GroupRowsArgs& g, int64_t s, int p0, int p1,
                                               int c0) {
  typedef float f32x4_t __attribute__((ext_vector_type(4)));
  const int l = lane_id();
  float acc[CH][8];
#pragma unroll
  for (int h = 0; h < CH; ++h)
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[h][k] = 0.f;
  bool on[CH];
#pragma unroll
  for (int h = 0; h < CH; ++h) on[h] = c0 + 512 * h + 8 * l < g.d;
  for (int b0 = p0; b0 < p1; b0 += kWave) {
    int e = 0;  // lane j: expert and activation of task b0 + j
    float av = 0.f;
    if (b0 + l < p1) {
      int32_t p = g.perm[b0 + l];
      p = p < 0 ? 0 : (p >= g.M ? (int32_t)(g.M - 1) : p);
      const int32_t ee = g.idx[p];
      e = ee < 0 ? 0 : (ee >= g.N ? (int)(g.N - 1) : ee);
      av = g.a[p];
    }
    const int nb = p1 - b0 < kWave ? p1 - b0 : kWave;
    for (int i = 0; i < nb; i += 4) {
      uint4 q[4][CH];
      float w4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool live = i + u < nb;  // wave-uniform
        const int ei = readlane_i32(e, live ? i + u : 0);
        w4[u] = live ? readlane_f32(av, i + u) : 0.f;
        const uint16_t* row = g.v + (int64_t)ei * g.d + c0 + 8 * l;
#pragma unroll
        for (int h = 0; h < CH; ++h)
          q[u][h] = (live && on[h]) ? *(const uint4*)(row + 512 * h) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int h = 0; h < CH; ++h) fma_bf16x8(acc[h], w4[u], q[u][h]);
    }
  }
#pragma unroll
  for (int h = 0; h < CH; ++h) {
    if (!on[h]) continue;
    // non-temporal: the rows are read once, by the sum, and must not evict the v rows
    float* o = g.rows + s * g.d + c0 + 512 * h + 8 * l;
    __builtin_nontemporal_store(f32x4_t{acc[h][0], acc[h][1], acc[h][2], acc[h][3]}, (f32x4_t*)o);
    __builtin_nontemporal_store(f32x4_t{acc[h][4], acc[h][5], acc[h][6], acc[h][7]},
                                (f32x4_t*)(o + 4));
  }
}

__global__ __launch_bounds__(kThreads) void group_rows_kernel(GroupRowsArgs g) {
  const int64_t n_slots = min((int64_t)g.counters[0], g.n_max);
  const int64_t waves = (int64_t)gridDim.x * (kThreads / kWave);
  const int64_t wv = xcd_contiguous(blockIdx.x, gridDim.x) * (kThreads / kWave) + (threadIdx.x >> 6);
  const int64_t per = (n_slots + waves - 1) / waves;
  const int64_t s_lo = wv * per;
  const int64_t s_hi = min(s_lo + per, n_slots);
  for (int64_t s = s_lo; s < s_hi; ++s) {
    const int p0 = g.slot_off[s], p1 = g.slot_off[s + 1];
    // the fp32 sums are the same whichever pass holds a column (each column is its own sum)
    int c0 = 0;
    for (; c0 + 2048 <= g.d; c0 += 2048) group_row_pass<4>(g, s, p0, p1, c0);
    if (g.d - c0 > 512) group_row_pass<4>(g, s, p0, p1, c0);
    else if (g.d > c0) group_row_pass<1>(g, s, p0, p1, c0);
  }
}

// y_t = sum of token t's slot rows, in group order (its run in the slot order). One wave per
// token.
struct SumRowsArgs {
  const float* rows;
  const int32_t* slots;
  const int32_t* tokens;
  const int32_t* tok_start;
  float* y;
  int64_t T, n;
  int d;
};

__global__ __launch_bounds__(kThreads) void sum_group_rows_kernel(SumRowsArgs g) {
  const int l = lane_id();
  const int64_t waves = (int64_t)gridDim.x * (kThreads / kWave);
  typedef float f32x4_t __attribute__((ext_vector_type(4)));
  for (int64_t t = (int64_t)blockIdx.x * (kThreads / kWave) + (threadIdx.x >> 6); t < g.T;
       t += waves) {
    const int i0 = g.tok_start[t];
    for (int c0 = 0; c0 < g.d; c0 += 512) {
      const int c = c0 + 8 * l;
      const bool on = c < g.d;
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (i0 >= 0) {
        for (int64_t b0 = i0;; b0 += kWave) {
          const int64_t i = b0 + l;
          const bool mine = i < g.n && g.tokens[i] == (int32_t)t;
          const int sl = mine ? g.slots[i] : 0;
          const int nb = __popcll(__ballot(mine));  // a prefix of the lanes: the run is contiguous
          for (int j = 0; j < nb; j += 4) {
            f32x4_t lo[4], hi[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const bool live = j + u < nb;  // wave-uniform
              const int sj = readlane_i32(sl, live ? j + u : 0);
              const float* r = g.rows + (int64_t)sj * g.d + c;
              lo[u] = (live && on) ? __builtin_nontemporal_load((const f32x4_t*)r) : f32x4_t{0.f, 0.f, 0.f, 0.f};
              hi[u] = (live && on) ? __builtin_nontemporal_load((const f32x4_t*)(r + 4)) : f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
            // added in slot order (u ascending), so the sum does not depend on the unrolling
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              acc[0] += lo[u].x; acc[1] += lo[u].y; acc[2] += lo[u].z; acc[3] += lo[u].w;
              acc[4] += hi[u].x; acc[5] += hi[u].y; acc[6] += hi[u].z; acc[7] += hi[u].w;
            }
          }
          if (nb < kWave) break;
        }
      }
      if (on) {
        float* o = g.y + t * g.d + c;
        __builtin_nontemporal_store(f32x4_t{acc[0], acc[1], acc[2], acc[3]}, (f32x4_t*)o);
        __builtin_nontemporal_store(f32x4_t{acc[4], acc[5], acc[6], acc[7]}, (f32x4_t*)(o + 4));
      }
    }
  }
}

}  // namespace

int grouped_tile_experts(int B) { return B <= 64 ? 64 : 160; }

hipError_t launch_grouped_dot(const Shape& s, const void* x, const void* u, const float* gates,
                              const int32_t* perm, const int32_t* active,
                              const int32_t* n_active, const GroupPlan& plan, float* a,
                              hipStream_t st) {
  if (s.M == 0) return hipSuccess;
  GroupedDotArgs g;
  g.x = (const uint16_t*)x;
  g.u = (const uint16_t*)u;
  g.gates = gates;
  g.perm = perm;
  g.active = active;
  g.n_active = n_active;
  g.slot_token = plan.slot_token;
  g.slot_off = plan.slot_off;
  g.key = plan.key;
  g.gbits = plan.gbits;
  g.grp_slot = plan.grp_slot;
  g.grp_tile = plan.grp_tile;
  g.counters = plan.counters;
  g.a = a;
  g.M = s.M;
  g.N = s.N;
  g.G = plan.G;
  g.d = s.d;
  g.B = s.B;
  g.act = s.act;
  // persistent: a multiple of eight workgroups, one or two per compute unit
  if (grouped_tile_experts(s.B) == 64)
    hipLaunchKernelGGL(grouped_dot_kernel<2>, dim3(512), dim3(kThreads),
                       2 * TileShape<2>::kStage, st, g);
  else
    hipLaunchKernelGGL(grouped_dot_kernel<5>, dim3(256), dim3(kThreads),
                       2 * TileShape<5>::kStage, st, g);
  return hipGetLastError();
}

hipError_t launch_group_rows(const Shape& s, const void* v, const int32_t* idx,
                             const int32_t* perm, const float* a, const GroupPlan& plan,
                             const SlotOrder& order, float* rows, int64_t n_slots_max, float* y,
                             hipStream_t st) {
  if (s.M == 0) return hipSuccess;
  GroupRowsArgs g;
  g.v = (const uint16_t*)v;
  g.idx = idx;
  g.perm = perm;
  g.a = a;
  g.slot_off = plan.slot_off;
  g.counters = plan.counters;
  g.rows = rows;
  g.M = s.M;
  g.N = s.N;
  g.n_max = n_slots_max;
  g.d = s.d;
  hipLaunchKernelGGL(group_rows_kernel, dim3(2048), dim3(kThreads), 0, st, g);
  SumRowsArgs r;
  r.rows = rows;
  r.slots = order.slots;
  r.tokens = order.tokens;
  r.tok_start = order.tok_start;
  r.y = y;
  r.T = s.T;
  r.n = n_slots_max;
  r.d = s.d;
  const int64_t wgs = (s.T + 3) / 4;
  hipLaunchKernelGGL(sum_group_rows_kernel, dim3((unsigned)(wgs < 8192 ? wgs : 8192)),
                     dim3(kThreads), 0, st, r);
  return hipGetLastError();
}

}  // namespace omnimoe
