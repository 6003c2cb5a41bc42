// Router logits (Eq. 9): one NT GEMM per grid half, C = Xq * Keys^T, where Xq is the
// token's query slice x[:, c0:c0+d_key] and Keys stacks the H heads' sub-key tables
// ([H * n_half, d_key]). Both operands are contiguous along d_key, so MFMA fragments load
// straight from row-major memory. The same kernels serve the dense router of the ablation
// (one half of N gating vectors), the shared MLP's projections (accumulating into y), the split-K
// second product of Eq. 14 over all experts and, with a masked-activation epilogue, its first
// product (x . u for every (token, expert) pair, g * act kept at the selected pairs only).
//
// bf16, d_key % 64 == 0: 256 x 256 tile, eight waves of 128 x 64 on v_mfma_f32_32x32x16_bf16,
//   operands copied global -> LDS without registers (two 64 KiB stages, XOR-swizzled rows);
// bf16, one to four tokens, d_key = 128 * 2^k <= 2048: sixteen lanes per key row with coalesced
//   loads and v_dot2_f32_bf16 (no MFMA);
// bf16, at most 64 tokens, d_key % 256 == 0: a split-K decode kernel with the token rows in LDS
//   (8 or more tokens, d_key <= 1024), else a split-K skinny kernel with operands straight from
//   memory;
// bf16 otherwise: 128 x 128 tile, four waves of 64 x 64 on v_mfma_f32_16x16x32_bf16, LDS
//   double buffer fed through registers;
// fp32: a VALU FMA tile kernel (the fp32 layer is small; fp32 MFMA would change rounding).
// All accumulate in fp32.
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct ScoreArgs {
  const void* x;
  const void* keys[2];
  float* out;
  int64_t T;
  int d;
  int dk;
  int H;
  int nh[2];        // rows per head of each half's key table
  int col0[2];      // first x column of each half's query
  int out_off[2];   // column offset of each half inside one (t, h) output row
  int per_head;     // nr + nc
  int64_t ldo;      // H * (nr + nc)
  // split-K (large kernel only): grid z is the split; split z covers k in [z kchunk, (z + 1)
  // kchunk) of half 0 and writes its partial product at out + z part_stride
  int kchunk;
  int64_t part_stride;
  // masked-activation epilogue (large kernel with ADOT): for token t and expert column n <
  // ncols_out, aout[t, n] = bf16(g * act(C[t, n])) when bit n of sel_mask[t] is set, where g is
  // the gate of that expert (sel_gates[t, rank], rank = selected experts of t below n), else 0
  const uint32_t* sel_mask;  // [T, words] bit n % 32 of word n / 32
  const int32_t* sel_pre;    // [T, words] selected experts of t in the words before
  const float* sel_gates;    // [T, hk] gates of t's selected experts in expert-id order
  uint16_t* aout;            // [T, ncols_out] bf16
  int64_t words;
  int ncols_out;
  int hk;
  int act;
};

// One output element (ACC: added to what is there). Each element is written by exactly one
// lane, so the sum is deterministic. ACC is a template parameter rather than a flag: with a
// runtime flag the compiler may hoist the read of out above the branch (the store makes the
// address safe to read), which would read every logit back.
template <bool ACC>
__device__ __forceinline__ void store_out(const ScoreArgs& a, int64_t off, float v) {
  if constexpr (ACC) a.out[off] += v;
  else a.out[off] = v;
}

// Output column of GEMM column n (head n / nh, key n % nh) within a token's row.
__device__ __forceinline__ int64_t out_col(const ScoreArgs& a, int half, int n) {
  int h = n / a.nh[half];
  int i = n - h * a.nh[half];
  return (int64_t)h * a.per_head + a.out_off[half] + i;
}

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_ROW = BK + 8;  // bf16 per LDS row: 144 B keeps 16-lane b128 reads conflict-free

template <bool ACC>
__global__ __launch_bounds__(256) void score_bf16_kernel(ScoreArgs a) {
  const int half = blockIdx.z;
  const int ncols = a.H * a.nh[half];
  const int n0 = blockIdx.x * BN;
  if (n0 >= ncols) return;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const uint16_t* X = (const uint16_t*)a.x;
  const uint16_t* Kt = (const uint16_t*)a.keys[half];
  const int c0 = a.col0[half];

  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDS_ROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;

  // Global-load assignment: chunk c = tid + 256 j (j < 4) is row c / 8, 16-byte column c % 8.
  uint4 ra[4], rb[4];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int c = tid + 256 * j;
      int r = c >> 3, kc = (c & 7) * 8;
      int64_t gm = m0 + r;
      int gn = n0 + r;
      bool kin = (k0 + kc) < a.dk;
      ra[j] = make_uint4(0, 0, 0, 0);
      rb[j] = make_uint4(0, 0, 0, 0);
      if (kin && gm < a.T) ra[j] = *(const uint4*)(X + gm * a.d + c0 + k0 + kc);
      if (kin && gn < ncols) rb[j] = *(const uint4*)(Kt + (int64_t)gn * a.dk + k0 + kc);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int c = tid + 256 * j;
      int r = c >> 3, kc = (c & 7) * 8;
      *(uint4*)(&As[buf][r * LDS_ROW + kc]) = ra[j];
      *(uint4*)(&Bs[buf][r * LDS_ROW + kc]) = rb[j];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = (a.dk + BK - 1) / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();

  // MFMA 16x16x32 operand layout: lane l holds row (l % 16) of A (column of B) and the
  // eight k values 8 * (l / 16) .. 8 * (l / 16) + 7.
  const int frag_row = lane & 15;
  const int frag_k = (lane >> 4) * 8;

  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) load_tile((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      bf16x8 fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int r = wm * 64 + i * 16 + frag_row;
        fa[i] = *(const bf16x8*)(&As[cur][r * LDS_ROW + ks + frag_k]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int r = wn * 64 + j * 16 + frag_row;
        fb[j] = *(const bf16x8*)(&Bs[cur][r * LDS_ROW + ks + frag_k]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) store_tile(cur ^ 1);
    __syncthreads();
  }

  // Accumulator layout: acc[i][j][r] is row 4 * (l / 16) + r, column l % 16 of the
  // 16x16 tile (i, j).
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int n = n0 + wn * 64 + j * 16 + (lane & 15);
    if (n >= ncols) continue;
    int64_t oc = out_col(a, half, n);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        int64_t m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
        if (m < a.T) store_out<ACC>(a, m * a.ldo + oc, acc[i][j][r]);
      }
    }
  }
}

// ---------------------------------------------------------------- large-tile bf16 kernel
// 256 x 256 macro tile, eight waves of 128 x 64 (4 x 2 MFMA tiles each; two waves per SIMD, so
// one wave's MFMAs run while the other waits for its LDS fragments or the barrier: 0.604 ->
// 0.587 ms at the training shape against four waves of 128 x 128, for 1.5x the LDS reads),
// k-step 64, two LDS stages filled straight from global memory (global_load_lds_dwordx4, no
// register staging). LDS rows are 128 B (64 bf16); the 16-byte chunk j of row r is stored at
// position j ^ ((r >> 1) & 7), so the 16 rows read by one MFMA operand load fall in distinct
// banks. Requires d_key % 64 == 0; tails in T and in the key count are handled by clamping the
// row that is loaded (those rows are never stored).

constexpr int LM = 256, LN = 256, LK = 64;
constexpr int LROW = LK * 2;                 // bytes per LDS row
constexpr int LSTAGE = (LM + LN) * LROW;      // bytes per stage: 64 KiB

typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Epilogue of the masked-activation product (the first product of Eq. 14 over all experts).
// Only the selected cells of a tile (a few percent in the layers that take this product) need
// the activation. The wave's 128 x 64 region of A is first cleared with 16-byte stores; then,
// a quarter (32 rows) at a time, the wave's accumulators are staged in LDS, each lane takes one
// selection word of the quarter (a row's 32 columns) and the wave queues the words' set bits,
// the k-th set bit of every lane in step k (a ballot places them), and the queued cells are
// evaluated on packed lanes, two per lane at a time so that their gate loads are in flight
// together, and stored over the cleared region (after a wait for the clearing stores). The work
// is then proportional to the words and the selected cells, not to the 8192 cells of the region.
// LDS (the operand stages are free by now): selection words and prefix counts of the tile's 256
// rows x 8 words (16 KiB); per wave a quarter of accumulators, [32 rows][65] fp32 (an odd row
// stride, so that the 4-byte staging stores of a half-wave hit distinct banks), and a queue of
// up to 2048 positions (4 KiB).
constexpr int kQRow = 65;

// The tile's selection words and prefix counts, four of each per thread (entry tid + 512 i is
// row (tid + 512 i) / 8, word (tid + 512 i) % 8 of the tile), loaded before the main loop so
// that their latency is hidden behind it.
struct TileSel {
  uint32_t w[4];
  int32_t p[4];
};

__device__ __forceinline__ TileSel load_tile_sel(const ScoreArgs& a, int64_t m0, int n0,
                                                 int tid) {
  TileSel ts;
  const int64_t w0 = n0 >> 5;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = tid + 512 * i;
    const int64_t t = m0 + (e >> 3), w = w0 + (e & 7);
    const bool ok = t < a.T && w < a.words;
    ts.w[i] = ok ? a.sel_mask[t * a.words + w] : 0u;
    ts.p[i] = ok ? a.sel_pre[t * a.words + w] : 0;
  }
  return ts;
}

__device__ __forceinline__ void act_mask_epilogue(const ScoreArgs& a, const f32x16 (&acc)[4][2],
                                                  const TileSel& ts, unsigned char* smem,
                                                  int64_t m0, int n0, int wm, int wn, int wid,
                                                  int lane, int tid) {
  uint32_t* lw = (uint32_t*)smem;                                   // [256][8]
  int32_t* lp = (int32_t*)(smem + 8192);                            // [256][8]
  float* R = (float*)(smem + 16384 + wid * (32 * kQRow * 4));       // [32][kQRow]
  uint16_t* qe = (uint16_t*)(smem + 16384 + 8 * (32 * kQRow * 4) + wid * 4096);  // [2048]
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    lw[tid + 512 * i] = ts.w[i];
    lp[tid + 512 * i] = ts.p[i];
  }
  __syncthreads();
  const int nw = n0 + wn * 64;  // first column of this wave's region (ncols_out % 64 == 0)
  if (nw >= a.ncols_out) return;
  // wave-uniform bases of the region's rows in A and in the gate table; offsets from them fit
  // in 32 bits (128 rows of at most 2^20 columns, or of hk <= 4096 gates)
  const int64_t t0 = m0 + wm * 128;
  uint16_t* const abase = a.aout + t0 * a.ncols_out + nw;
  const float* const gbase = a.sel_gates + t0 * a.hk;
  const int ldo = a.ncols_out, hk = a.hk;
  {
    const int nrows = a.T - t0 < 128 ? (int)(a.T - t0) : 128;
    const uint4 z = make_uint4(0, 0, 0, 0);
#pragma unroll 4
    for (int rr = lane >> 3; rr < nrows; rr += 8) *(uint4*)(abase + rr * ldo + (lane & 7) * 8) = z;
  }
  bool cleared = false;  // the clearing stores have completed
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // stage: lane (c, h) holds column j 32 + c, row 8 (q / 4) + 4 h + q % 4 in acc[i][j][q]
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int r = (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        R[r * kQRow + j * 32 + (lane & 31)] = acc[i][j][q];
      }
    // this lane's word: row lane / 2 of the quarter, columns (lane % 2) 32 .. + 31
    uint32_t w = lw[(wm * 128 + i * 32 + (lane >> 1)) * 8 + wn * 2 + (lane & 1)];
    int total = 0;
    for (uint64_t b = __ballot(w != 0u); b; b = __ballot(w != 0u)) {
      if (w) {
        const int pos = total + __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32),
                                                          __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0));
        const int bit = __builtin_ctz(w);
        w &= w - 1u;
        qe[pos] = (uint16_t)(((lane >> 1) << 6) | ((lane & 1) * 32 + bit));
      }
      total += __popcll(b);
    }
    wave_lds_sync();
    if (total > 0 && !cleared) {
      wait_vm0();
      cleared = true;
    }
    // Two entries per lane at a time; entries past total read the last entry again (unguarded
    // loads stay in flight together) and store nothing.
    for (int base = 0; base < total; base += 2 * kWave) {
      float h[2], gt[2];
      int o[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int k = base + u * kWave + lane < total ? base + u * kWave + lane : total - 1;
        const int e = qe[k];
        const int rq = e >> 6, cc = e & 63;
        h[u] = R[rq * kQRow + cc];
        const int rw = i * 32 + rq;  // row within the wave's region
        const int wi = (wm * 128 + rw) * 8 + wn * 2 + (cc >> 5);
        const int rank = lp[wi] + __popc(lw[wi] & ((1u << (cc & 31)) - 1u));
        gt[u] = gbase[rw * hk + rank];
        o[u] = rw * ldo + cc;
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
        if (base + u * kWave + lane < total)
          abase[o[u]] = bf16_rne(gt[u] * activation(a.act, h[u]));
    }
    wave_lds_sync();
  }
}

template <bool ACC, bool SPLIT = false, bool ADOT = false>
__global__ __launch_bounds__(512, 1) void score_bf16_large_kernel(ScoreArgs a) {
  const int half = SPLIT ? 0 : blockIdx.z;
  const int ncols = a.H * a.nh[half];
  int tile_n = blockIdx.x, tile_m = blockIdx.y;
  if constexpr (ADOT) {
    // One-dimensional grid. Workgroup b runs on XCD b % 8; each XCD takes a contiguous range of
    // tiles in column-major order, so the token-row tiles that share an expert tile run together
    // on one XCD and that tile of U is fetched into its L2 once.
    const int ntm = (int)((a.T + LM - 1) / LM);
    const int total = ((a.ncols_out + LN - 1) / LN) * ntm;
    const int per = (total + 7) / 8;
    const int k = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
    if (k >= total || (int)(blockIdx.x / 8) >= per) return;
    tile_n = k / ntm;
    tile_m = k - tile_n * ntm;
  }
  const int n0 = tile_n * LN;
  if (n0 >= (ADOT ? a.ncols_out : ncols)) return;
  const int64_t m0 = (int64_t)tile_m * LM;
  const int64_t kbase = SPLIT ? (int64_t)blockIdx.z * a.kchunk : 0;
  const uint16_t* X = (const uint16_t*)a.x + kbase;
  const uint16_t* Kt = (const uint16_t*)a.keys[half] + kbase;
  const int c0 = a.col0[half];
  [[maybe_unused]] float* const out = SPLIT ? a.out + (int64_t)blockIdx.z * a.part_stride : a.out;

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int wm = wid >> 2, wn = wid & 3;

  // Loader: instruction i (0..3) of wave w covers rows 8 (4 w + i) .. +8 of A and of B; lane l
  // fills LDS position l % 8 of row l / 8, i.e. global chunk (l % 8) ^ swz(row).
  const uint16_t* ga[4];
  const uint16_t* gb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = (wid * 4 + i) * 8 + (lane >> 3);
    const int j = (lane & 7) ^ swz(r);
    int64_t gm = m0 + r;
    if (gm >= a.T) gm = a.T - 1;
    int gn = n0 + r;
    if (gn >= ncols) gn = ncols - 1;
    ga[i] = X + gm * a.d + c0 + j * 8;
    gb[i] = Kt + (int64_t)gn * a.dk + j * 8;
  }
  auto issue = [&](int stage, int k0) {
    unsigned char* base = smem + stage * LSTAGE;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      unsigned char* la = base + (wid * 4 + i) * 8 * LROW;
      unsigned char* lb = base + LM * LROW + (wid * 4 + i) * 8 * LROW;
      __builtin_amdgcn_global_load_lds((const void*)(ga[i] + k0), (lds_ptr_t)la, 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(gb[i] + k0), (lds_ptr_t)lb, 16, 0, 0);
    }
  };

  // v_mfma_f32_32x32x16_bf16: lane l holds row (l % 32) of the A operand (column of B) and k
  // values 8 (l / 32) .. +7 of a 16-wide k step; accumulator register q of a 32 x 32 tile is
  // row 8 (q / 4) + 4 (l / 32) + q % 4, column l % 32.
  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

  const int KT = (SPLIT ? a.kchunk : a.dk) / LK;
  [[maybe_unused]] TileSel sel;
  if constexpr (ADOT) sel = load_tile_sel(a, m0, n0, tid);
  issue(0, 0);
  wait_vm0();
  __syncthreads();

  const int frow = lane & 31;
  const int fk = lane >> 5;  // 16-byte chunk within a 16-wide k step
  int a_off[4], b_off[4];    // LDS row offsets of this lane's operand rows
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a_off[i] = (wm * 128 + i * 32 + frow) * LROW;
    b_off[i] = LM * LROW + (wn * 64 + (i & 1) * 32 + frow) * LROW;
  }
  const int sw = swz(frow);  // rows i * 32 + frow share (r >> 1) & 7 with frow
  auto frag = [&](const unsigned char* st, int off, int ks) -> bf16x8 {
    return *(const bf16x8*)(st + off + (((ks * 2 + fk) ^ sw) << 4));
  };
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) issue(cur ^ 1, (kt + 1) * LK);
    const unsigned char* st = smem + cur * LSTAGE;
    bf16x8 fa[2][4], fb[2][2];
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[0][i] = frag(st, a_off[i], 0);
#pragma unroll
    for (int i = 0; i < 2; ++i) fb[0][i] = frag(st, b_off[i], 0);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int c = ks & 1;
      if (ks + 1 < 4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[c ^ 1][i] = frag(st, a_off[i], ks + 1);
#pragma unroll
        for (int i = 0; i < 2; ++i) fb[c ^ 1][i] = frag(st, b_off[i], ks + 1);
      }
      // keep the double buffer: the next step's fragment reads are issued before this step's
      // MFMAs (left alone, the scheduler sinks each read next to its use)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[c][i], fb[c][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    wait_vm0();
    __syncthreads();
  }

  // Epilogue. Each lane writes column n of rows m_lane + r, r = i * 32 + 8 (q / 4) + q % 4:
  // one row pointer per column block and compile-time row offsets times the uniform stride.
  // Only a tile that reaches past T checks rows, with one tile-wide branch; a per-element
  // check costs a divergent branch per store, which made the epilogue as long as a quarter
  // of the main loop.
  if constexpr (ADOT) {
    act_mask_epilogue(a, acc, sel, smem, m0, n0, wm, wn, wid, lane, tid);
    return;
  }
  const int64_t m_lane = m0 + wm * 128 + (lane >> 5) * 4;
  float* const obase = SPLIT ? out : a.out;
  auto store_all = [&](auto rows_ok) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn * 64 + j * 32 + (lane & 31);
      if (n >= ncols) continue;
      float* const orow = obase + m_lane * a.ldo + out_col(a, half, n);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int r = i * 32 + (q >> 2) * 8 + (q & 3);
          if (!rows_ok(r)) continue;
          float* const o = orow + (int64_t)r * a.ldo;
          if constexpr (SPLIT) *o = acc[i][j][q];
          else if constexpr (ACC) *o += acc[i][j][q];
          // non-temporal: the next kernel reads these once, and dirty lines left in L2 would
          // otherwise be written back while it streams them
          else __builtin_nontemporal_store(acc[i][j][q], o);
        }
      }
    }
  };
  if (m0 + LM <= a.T) store_all([](int) { return true; });
  else store_all([&](int r) { return m_lane + r < a.T; });
}

// ---------------------------------------------------------------- few-token bf16 kernel
// For T <= 4: reading the sub-keys once is the whole cost, and MFMA fragments (32 rows x 32
// bytes per load instruction) make the loads address-bound. Here sixteen lanes share a key row
// and read it in coalesced 256-byte pieces (lane c of the sixteen takes chunks c, c + 16, ...
// of 8 bf16), each lane forming TT partial dot products with v_dot2_f32_bf16 against the token
// rows held in registers; the sixteen partial sums of a (token, key) pair are added in a fixed
// tree (DPP within each 16-lane row). A wave covers four keys, a workgroup of four waves
// sixteen. Requires d_key = 128 CH with CH = 1, 2, 4, 8 or 16.
constexpr int GV_KEYS = 16;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// v_dot2_f32_bf16 on two words of bf16 pairs. The words are taken by value: a bit cast applied
// straight to an element of a vector (v.y) has been seen to compile to the cast of element 0.
__device__ __forceinline__ float dot2_words(uint32_t p, uint32_t q, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, p),
                                         __builtin_bit_cast(bf16x2_t, q), acc, false);
}

template <bool ACC, int TT, int CH>
__global__ __launch_bounds__(256) void score_bf16_gemv_kernel(ScoreArgs a) {
  const int half = blockIdx.y;
  const int ncols = a.H * a.nh[half];
  // a workgroup past the half's keys (all of them for an empty half, as the shared MLP's and the
  // dense router's single-half products have) reads nothing: the clamp below needs a key
  if ((int)blockIdx.x * GV_KEYS >= ncols) return;
  const int lane = threadIdx.x & 63, c16 = lane & 15;
  const int n = blockIdx.x * GV_KEYS + (threadIdx.x >> 4);  // this row of sixteen lanes' key
  const int nn = n < ncols ? n : ncols - 1;
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4* kr = (const u32x4*)((const uint16_t*)a.keys[half] + (int64_t)nn * a.dk) + c16;
  u32x4 kv[CH];
#pragma unroll
  for (int q = 0; q < CH; ++q) kv[q] = __builtin_nontemporal_load(kr + 16 * q);
  __builtin_amdgcn_sched_barrier(0);  // every key load is issued before the first use
  float acc[TT];
#pragma unroll
  for (int t = 0; t < TT; ++t) {
    const u32x4* xr = (const u32x4*)((const uint16_t*)a.x + (int64_t)(t < a.T ? t : a.T - 1) * a.d +
                                     a.col0[half]) + c16;
    float s = 0.0f;
#pragma unroll
    for (int q = 0; q < CH; ++q) {
      const u32x4 xv = xr[16 * q];
      s = dot2_words(kv[q].x, xv.x, s);
      s = dot2_words(kv[q].y, xv.y, s);
      s = dot2_words(kv[q].z, xv.z, s);
      s = dot2_words(kv[q].w, xv.w, s);
    }
    // sum over the sixteen lanes of the row (quad swaps, then rotations by 4 and 8)
    int x = __float_as_int(s);
    s += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));
    x = __float_as_int(s);
    s += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));
    x = __float_as_int(s);
    s += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x124, 0xF, 0xF, false));
    x = __float_as_int(s);
    s += __int_as_float(__builtin_amdgcn_update_dpp(x, x, 0x128, 0xF, 0xF, false));
    acc[t] = s;
  }
  if (n < ncols) {
    const int64_t oc = out_col(a, half, n);
#pragma unroll
    for (int t = 0; t < TT; ++t)
      if (c16 == t && t < a.T) store_out<ACC>(a, (int64_t)t * a.ldo + oc, acc[t]);
  }
}

// ---------------------------------------------------------------- skinny bf16 kernel
// For T <= 64 (decode): the work is reading the sub-keys once. A workgroup owns 32 keys of one
// half for all (<= 64) tokens; its four waves split d_key in four quarters, load MFMA operand
// fragments straight from global memory (no LDS staging), and run v_mfma_f32_32x32x16_bf16 on
// a 32·RB x 32 tile each (RB = 1 row block when T <= 32, else 2); the four partial tiles are then
// added through LDS in wave order, so the sum order is fixed. Requires d_key % 256 == 0 (each
// wave's quarter is a multiple of 64).

constexpr int SK_N = 32;

// STEPS > 0: d_key = 64 STEPS, and all STEPS fragment pairs of the wave's quarter are requested
// at once; STEPS = 0: any d_key % 256 == 0, four k steps in flight per iteration.
template <bool ACC, int RB, int STEPS>
__global__ __launch_bounds__(256) void score_bf16_skinny_kernel(ScoreArgs a) {
  const int half = blockIdx.y;
  const int ncols = a.H * a.nh[half];
  const int n0 = blockIdx.x * SK_N;
  if (n0 >= ncols) return;
  const uint16_t* X = (const uint16_t*)a.x + a.col0[half];
  const uint16_t* Kt = (const uint16_t*)a.keys[half];
  __shared__ float part[3][64 * SK_N];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int kq = a.dk / 4;  // this wave's k range: [wid * kq, (wid + 1) * kq)
  const int frow = lane & 31, fk = (lane >> 5) * 8;
  // operand rows: tokens 0..63 (clamped to T - 1) and keys n0 .. n0 + 63 (clamped)
  const uint16_t* pa[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    int64_t m = i * 32 + frow;
    if (m >= a.T) m = a.T - 1;
    pa[i] = X + m * a.d + wid * kq + fk;
  }
  int n = n0 + frow;
  if (n >= ncols) n = ncols - 1;
  const uint16_t* pb = Kt + (int64_t)n * a.dk + wid * kq + fk;
  f32x16 acc[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[i][q] = 0.f;
  if constexpr (STEPS > 0) {
    bf16x8 fa[STEPS][RB], fb[STEPS];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
#pragma unroll
      for (int i = 0; i < RB; ++i) fa[s][i] = *(const bf16x8*)(pa[i] + 16 * s);
      fb[s] = *(const bf16x8*)(pb + 16 * s);
    }
    __builtin_amdgcn_sched_barrier(0);  // keeps every load ahead of the first MFMA
#pragma unroll
    for (int s = 0; s < STEPS; ++s)
#pragma unroll
      for (int i = 0; i < RB; ++i)
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s], acc[i], 0, 0, 0);
  } else {
    // four k steps of 16 in flight per iteration
    for (int k = 0; k < kq; k += 64) {
      bf16x8 fa[4][RB], fb[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int i = 0; i < RB; ++i) fa[s][i] = *(const bf16x8*)(pa[i] + k + 16 * s);
        fb[s] = *(const bf16x8*)(pb + k + 16 * s);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < RB; ++i)
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s][i], fb[s], acc[i], 0, 0, 0);
    }
  }
  // tile element (row, col) of a 32 x 32 block: register q, lane l with
  // row = 8 (q / 4) + 4 (l / 32) + q % 4, col = l % 32
  const int c = lane & 31;
  if (wid > 0) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int r = i * 32 + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        part[wid - 1][r * SK_N + c] = acc[i][q];
      }
  }
  __syncthreads();
  if (wid == 0 && n0 + c < ncols) {
    const int64_t oc = out_col(a, half, n0 + c);
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int r = i * 32 + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        const float v = ((acc[i][q] + part[0][r * SK_N + c]) + part[1][r * SK_N + c]) +
                        part[2][r * SK_N + c];
        if (r < a.T) store_out<ACC>(a, (int64_t)r * a.ldo + oc, v);
      }
  }
}

// ---------------------------------------------------------------- decode bf16 kernel
// For T <= 64 and d_key <= 1024 (decode): a workgroup owns 64 keys of one half. Four copy
// waves put the half's token rows (32·RB rows of d_key, RB = 1 when T <= 32, else 2) into LDS
// with coalesced 16-byte loads, while eight compute waves request their key
// fragments: wave w takes key block w % 2 (32 keys) over quarter w / 2 of d_key, STEPS
// fragments, all in flight at once. After one barrier the compute waves run
// v_mfma_f32_32x32x16_bf16 step by step as their fragments arrive, with the token fragments
// read from LDS (the copy runs on other waves, so no compute wave waits for it through its own
// load counter; it goes through registers, since an LDS read after a direct-to-LDS load makes
// the compiler wait for every outstanding load, the fragments included). The four quarters' partial tiles go through LDS and every compute thread adds
// four of them in quarter order (the sum order is fixed) and stores its share of the
// 32·RB x 64 tile. LDS row r holds its 16-byte chunk c at c ^ (r % 16) within each group of
// sixteen, so the sixteen rows read by a quarter-wave fall in distinct banks. Requires
// d_key % 256 == 0.

constexpr int DC_KEYS = 64;
constexpr int DC_WAVES = 8;       // compute waves
constexpr int DC_COPY_WAVES = 4;  // token-copy waves

size_t decode_lds_bytes(int dk, int rb) {
  const size_t xb = (size_t)rb * 32 * dk * 2;                 // token rows
  const size_t pb = (size_t)8 * rb * 32 * 32 * sizeof(float);  // partial tiles of the quarters
  return xb > pb ? xb : pb;
}

template <bool ACC, int RB, int STEPS>
__global__ __launch_bounds__(64 * (DC_WAVES + DC_COPY_WAVES)) void score_bf16_decode_kernel(
    ScoreArgs a) {
  const int half = blockIdx.y;
  const int ncols = a.H * a.nh[half];
  const int n0 = blockIdx.x * DC_KEYS;
  if (n0 >= ncols) return;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const uint16_t* X = (const uint16_t*)a.x + a.col0[half];
  const uint16_t* Kt = (const uint16_t*)a.keys[half];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int kb = wid & 1, qi = (wid >> 1) & 3;
  constexpr int kq = STEPS * 16;  // d_key / 4
  constexpr int dk = 4 * kq;
  constexpr int cpr = dk / 8;     // 16-byte chunks per token row
  constexpr int npos = RB * 32 * cpr;
  constexpr int per_wave = npos / (kWave * DC_COPY_WAVES);  // copy loads per copy wave
  static_assert(npos % (kWave * DC_COPY_WAVES) == 0, "the copy divides evenly");
  const int frow = lane & 31;
  bf16x8 fb[STEPS];
  // Both roles pass the same two barriers: the first once the copy's loads are issued (so the
  // compute unit's memory pipeline takes them ahead of the key fragments), the second once the
  // token rows are in LDS. The roles sit in separate branches up to the MFMAs, so the compute
  // waves' LDS reads never follow a direct-to-LDS load in program order (the compiler would
  // make them wait for every outstanding load, the key fragments included).
  f32x16 acc[RB];
#pragma unroll
  for (int i = 0; i < RB; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;
  if (wid >= DC_WAVES) {
    // token rows into LDS: 16-byte position p holds row p / cpr, chunk (p % cpr) ^ (row % 16)
    const int cw = wid - DC_WAVES;
#pragma unroll
    for (int j = 0; j < per_wave; ++j) {
      const int q = cw + DC_COPY_WAVES * j;
      const int p = q * kWave + lane;
      const int r = p / cpr;
      const int c = (p - r * cpr) ^ (r & 15);
      const int64_t m = r < a.T ? r : a.T - 1;
      __builtin_amdgcn_global_load_lds((const void*)(X + m * a.d + c * 8),
                                       (lds_ptr_t)(smem + (size_t)q * kWave * 16), 16, 0, 0);
    }
    __builtin_amdgcn_s_barrier();
    wait_vm0();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
  } else {
    __builtin_amdgcn_s_barrier();
    // this wave's key fragments, all in flight
    bf16x8 fb[STEPS];
    int n = n0 + kb * 32 + frow;
    if (n >= ncols) n = ncols - 1;
    const uint16_t* pb = Kt + (int64_t)n * dk + qi * kq + (lane >> 5) * 8;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) fb[s] = *(const bf16x8*)(pb + 16 * s);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();  // the token rows are in LDS
    asm volatile("" ::: "memory");
    const int c0 = qi * kq / 8 + (lane >> 5);  // logical chunk of step 0
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
#pragma unroll
      for (int i = 0; i < RB; ++i) {
        const int r = i * 32 + frow;
        const int ph = (c0 + 2 * s) ^ (r & 15);
        const bf16x8 fa = *(const bf16x8*)(smem + ((size_t)r * cpr + ph) * 16);
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb[s], acc[i], 0, 0, 0);
      }
    }
  }
  __syncthreads();  // the token rows are no longer needed: the space takes the partial tiles
  float* part = (float*)smem;  // [quarter][key block][32 RB rows][32 keys]
  if (wid < DC_WAVES) {
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
        part[((qi * 2 + kb) * RB * 32 + r) * 32 + (lane & 31)] = acc[i][e];
      }
  }
  __syncthreads();
  if (wid >= DC_WAVES) return;
  // thread t: keys 4 k4 .. 4 k4 + 3 of the tile's 64 (k4 = t % 16) in rows t / 16 + 32 j
  const int k4 = tid & 15;
  const int b = k4 >> 3, cc = (k4 & 7) * 4;
  const int nn0 = n0 + b * 32 + cc;
  int64_t col[4];
  {
    int h = nn0 / a.nh[half], i = nn0 - h * a.nh[half];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      col[t] = (int64_t)h * a.per_head + a.out_off[half] + i;
      if (++i == a.nh[half]) {
        i = 0;
        ++h;
      }
    }
  }
  // one 16-byte store when the four columns are consecutive and aligned
  const bool vec = nn0 + 3 < ncols && col[3] == col[0] + 3 && ((col[0] | a.ldo) & 3) == 0 &&
                   ((uintptr_t)a.out & 15) == 0;
#pragma unroll
  for (int j = 0; j < RB; ++j) {
    const int r = (j * 64 * DC_WAVES + tid) >> 4;
    float4 v = *(const float4*)&part[((0 * 2 + b) * RB * 32 + r) * 32 + cc];
#pragma unroll
    for (int qq = 1; qq < 4; ++qq) {
      const float4 w = *(const float4*)&part[((qq * 2 + b) * RB * 32 + r) * 32 + cc];
      v.x += w.x;
      v.y += w.y;
      v.z += w.z;
      v.w += w.w;
    }
    if (r >= a.T) continue;
    float* o = a.out + (int64_t)r * a.ldo;
    if (vec) {
      float4* o4 = (float4*)(o + col[0]);
      if constexpr (ACC) {
        const float4 w = *o4;
        v.x = w.x + v.x;
        v.y = w.y + v.y;
        v.z = w.z + v.z;
        v.w = w.w + v.w;
      }
      *o4 = v;
    } else {
      const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (nn0 + t < ncols) store_out<ACC>(a, (int64_t)r * a.ldo + col[t], vv[t]);
    }
  }
}

constexpr int FT = 64, FK = 16;

template <bool ACC>
__global__ __launch_bounds__(256) void score_f32_kernel(ScoreArgs a) {
  const int half = blockIdx.z;
  const int ncols = a.H * a.nh[half];
  const int n0 = blockIdx.x * FT;
  if (n0 >= ncols) return;
  const int64_t m0 = (int64_t)blockIdx.y * FT;
  const float* X = (const float*)a.x;
  const float* Kt = (const float*)a.keys[half];
  const int c0 = a.col0[half];
  __shared__ float As[FK][FT + 4], Bs[FK][FT + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.dk; k0 += FK) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int c = tid + 256 * j;
      int r = c >> 4, kk = c & 15;
      int64_t gm = m0 + r;
      int gn = n0 + r;
      bool kin = (k0 + kk) < a.dk;
      As[kk][r] = (kin && gm < a.T) ? X[gm * a.d + c0 + k0 + kk] : 0.f;
      Bs[kk][r] = (kin && gn < ncols) ? Kt[(int64_t)gn * a.dk + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int n = n0 + tx * 4 + j;
    if (n >= ncols) continue;
    int64_t oc = out_col(a, half, n);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int64_t m = m0 + ty * 4 + i;
      if (m < a.T) store_out<ACC>(a, m * a.ldo + oc, acc[i][j]);
    }
  }
}

}  // namespace

// Reads the GEMM's operands once, in 16-byte chunks, so that they sit in the memory-side cache
// (MALL, 256 MB) when the GEMM fetches them: the GEMM's two-stage pipeline covers the MALL's
// latency but not HBM's, and its tiles fetch every operand line several times from beyond
// L2. Three segments (x, row keys, column keys) in one grid-stride walk; nothing is written
// (the sink store cannot happen: it needs a negative count).
struct PrefetchArgs {
  const uint4* p[3];
  int64_t n[3];  // chunks per segment
  uint32_t* sink;
};

__global__ __launch_bounds__(256) void prefetch_kernel(PrefetchArgs a) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * 256;
#pragma unroll
  for (int seg = 0; seg < 3; ++seg) {
    const uint4* __restrict__ p = a.p[seg];
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < a.n[seg]; i += stride) {
      const uint4 v = p[i];
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  }
  if (acc == 0x9E3779B9u && a.n[0] < 0) *a.sink = acc;
}

constexpr int64_t kPrefetchMaxBytes = 128ll << 20;  // half the MALL

hipError_t launch_score(const Shape& s, const void* x, const void* keys_row,
                        const void* keys_col, float* half_scores, hipStream_t st,
                        bool accumulate) {
  ScoreArgs a;
  a.x = x;
  a.keys[0] = keys_row;
  a.keys[1] = keys_col;
  a.out = half_scores;
  a.T = s.T;
  a.d = s.d;
  a.dk = s.dk;
  a.H = s.H;
  a.nh[0] = s.nr;
  a.nh[1] = s.nc;
  a.col0[0] = 0;
  a.col0[1] = s.col0;
  a.out_off[0] = 0;
  a.out_off[1] = s.nr;
  a.per_head = s.nr + s.nc;
  a.ldo = (int64_t)s.H * (s.nr + s.nc);
  a.kchunk = 0;
  a.part_stride = 0;
  const int ncols = s.H * (s.nr > s.nc ? s.nr : s.nc);
  // (not for the accumulating product: its operand was just written and is in the caches)
  const bool large = s.bf16 && s.T > 64 && s.dk % 64 == 0;
  if (large && !accumulate) {
    // x rows are read whole (both query halves); the tables are [H, n, d_key] bf16
    PrefetchArgs pa;
    pa.p[0] = (const uint4*)x;
    pa.p[1] = (const uint4*)keys_row;
    pa.p[2] = (const uint4*)keys_col;
    pa.n[0] = s.T * s.d * 2 / 16;
    pa.n[1] = (int64_t)s.H * s.nr * s.dk * 2 / 16;
    pa.n[2] = (int64_t)s.H * s.nc * s.dk * 2 / 16;
    pa.sink = (uint32_t*)half_scores;
    if ((pa.n[0] + pa.n[1] + pa.n[2]) * 16 <= kPrefetchMaxBytes)
      hipLaunchKernelGGL(prefetch_kernel, dim3(4096), dim3(256), 0, st, pa);
  }
  if (s.bf16 && s.T >= 8 && s.T <= 64 && s.dk % 256 == 0 && s.dk <= 1024) {
    dim3 grid((ncols + DC_KEYS - 1) / DC_KEYS, 2);
    const int rb = s.T > 32 ? 2 : 1;
    const size_t lds = decode_lds_bytes(s.dk, rb);
    const dim3 block(64 * (DC_WAVES + DC_COPY_WAVES));
#define OMNIMOE_DECODE(ACC_, RB_, ST_) \
  hipLaunchKernelGGL((score_bf16_decode_kernel<ACC_, RB_, ST_>), grid, block, lds, st, a)
#define OMNIMOE_DECODE_STEPS(ACC_, RB_)                  \
  do {                                                   \
    switch (s.dk / 64) {                                 \
      case 4: OMNIMOE_DECODE(ACC_, RB_, 4); break;       \
      case 8: OMNIMOE_DECODE(ACC_, RB_, 8); break;       \
      case 12: OMNIMOE_DECODE(ACC_, RB_, 12); break;     \
      default: OMNIMOE_DECODE(ACC_, RB_, 16); break;     \
    }                                                    \
  } while (0)
    if (accumulate && rb == 2) OMNIMOE_DECODE_STEPS(true, 2);
    else if (accumulate) OMNIMOE_DECODE_STEPS(true, 1);
    else if (rb == 2) OMNIMOE_DECODE_STEPS(false, 2);
    else OMNIMOE_DECODE_STEPS(false, 1);
#undef OMNIMOE_DECODE_STEPS
#undef OMNIMOE_DECODE
  } else if (s.bf16 && s.T <= 4 && s.dk % 128 == 0 && s.dk <= 2048 &&
             ((s.dk / 128) & (s.dk / 128 - 1)) == 0) {
    const dim3 grid((ncols + GV_KEYS - 1) / GV_KEYS, 2);
#define OMNIMOE_GEMV(ACC_, TT_, CH_) \
  hipLaunchKernelGGL((score_bf16_gemv_kernel<ACC_, TT_, CH_>), grid, dim3(256), 0, st, a)
#define OMNIMOE_GEMV_CH(ACC_, TT_)                                           \
  do {                                                                       \
    const int ch = s.dk / 128;                                               \
    if (ch == 1) OMNIMOE_GEMV(ACC_, TT_, 1);                                 \
    else if (ch == 2) OMNIMOE_GEMV(ACC_, TT_, 2);                            \
    else if (ch == 4) OMNIMOE_GEMV(ACC_, TT_, 4);                            \
    else if (ch == 8) OMNIMOE_GEMV(ACC_, TT_, 8);                            \
    else OMNIMOE_GEMV(ACC_, TT_, 16);                                        \
  } while (0)
    if (accumulate) {
      if (s.T == 1) OMNIMOE_GEMV_CH(true, 1);
      else if (s.T == 2) OMNIMOE_GEMV_CH(true, 2);
      else OMNIMOE_GEMV_CH(true, 4);
    } else {
      if (s.T == 1) OMNIMOE_GEMV_CH(false, 1);
      else if (s.T == 2) OMNIMOE_GEMV_CH(false, 2);
      else OMNIMOE_GEMV_CH(false, 4);
    }
#undef OMNIMOE_GEMV_CH
#undef OMNIMOE_GEMV
  } else if (s.bf16 && s.T <= 64 && s.dk % 256 == 0) {
    dim3 grid((ncols + SK_N - 1) / SK_N, 2);
    // every fragment in flight at once for d_key <= 1024 (below 8 tokens: one row block)
    const int steps = s.dk <= 1024 ? s.dk / 64 : 0;
#define OMNIMOE_SKINNY(ACC_, RB_, ST_) \
  hipLaunchKernelGGL((score_bf16_skinny_kernel<ACC_, RB_, ST_>), grid, dim3(256), 0, st, a)
#define OMNIMOE_SKINNY_STEPS(ACC_, RB_)                  \
  do {                                                   \
    switch (steps) {                                     \
      case 4: OMNIMOE_SKINNY(ACC_, RB_, 4); break;       \
      case 8: OMNIMOE_SKINNY(ACC_, RB_, 8); break;       \
      case 12: OMNIMOE_SKINNY(ACC_, RB_, 12); break;     \
      case 16: OMNIMOE_SKINNY(ACC_, RB_, 16); break;     \
      default: OMNIMOE_SKINNY(ACC_, RB_, 0); break;      \
    }                                                    \
  } while (0)
    if (accumulate && s.T > 32) OMNIMOE_SKINNY(true, 2, 0);
    else if (accumulate) OMNIMOE_SKINNY(true, 1, 0);
    else if (s.T > 32) OMNIMOE_SKINNY(false, 2, 0);
    else if (s.T > 8) OMNIMOE_SKINNY(false, 1, 0);
    else OMNIMOE_SKINNY_STEPS(false, 1);
#undef OMNIMOE_SKINNY_STEPS
#undef OMNIMOE_SKINNY
  } else if (s.bf16 && s.dk % LK == 0) {
    dim3 grid((ncols + LN - 1) / LN, (unsigned)((s.T + LM - 1) / LM), 2);
    if (accumulate)
      hipLaunchKernelGGL(score_bf16_large_kernel<true>, grid, dim3(512), 2 * LSTAGE, st, a);
    else
      hipLaunchKernelGGL(score_bf16_large_kernel<false>, grid, dim3(512), 2 * LSTAGE, st, a);
  } else if (s.bf16) {
    dim3 grid((ncols + BN - 1) / BN, (unsigned)((s.T + BM - 1) / BM), 2);
    if (accumulate)
      hipLaunchKernelGGL(score_bf16_kernel<true>, grid, dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(score_bf16_kernel<false>, grid, dim3(256), 0, st, a);
  } else {
    dim3 grid((ncols + FT - 1) / FT, (unsigned)((s.T + FT - 1) / FT), 2);
    if (accumulate)
      hipLaunchKernelGGL(score_f32_kernel<true>, grid, dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL(score_f32_kernel<false>, grid, dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_splitk(int64_t M, int N, const void* A, int64_t lda, const void* B,
                              int64_t ldb, int kchunk, int splits, float* out, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  ScoreArgs a;
  a.x = A;
  a.keys[0] = B;
  a.keys[1] = B;
  a.out = out;
  a.T = M;
  a.d = (int)lda;
  a.dk = (int)ldb;
  a.H = 1;
  a.nh[0] = N;
  a.nh[1] = 0;
  a.col0[0] = 0;
  a.col0[1] = 0;
  a.out_off[0] = 0;
  a.out_off[1] = 0;
  a.per_head = N;
  a.ldo = N;
  a.kchunk = kchunk;
  a.part_stride = M * (int64_t)N;
  dim3 grid((N + LN - 1) / LN, (unsigned)((M + LM - 1) / LM), splits);
  hipLaunchKernelGGL((score_bf16_large_kernel<false, true>), grid, dim3(512), 2 * LSTAGE, st, a);
  return hipGetLastError();
}

hipError_t launch_gemm_act_mask(int64_t T, int N, int ncols_out, const void* x, int d,
                                const void* u, const uint32_t* sel_mask, const int32_t* sel_pre,
                                int64_t words, const float* sel_gates, int hk, int act,
                                uint16_t* aout, hipStream_t st) {
  if (T == 0 || ncols_out == 0) return hipSuccess;
  ScoreArgs a = {};
  a.x = x;
  a.keys[0] = u;
  a.keys[1] = u;
  a.out = nullptr;
  a.T = T;
  a.d = d;
  a.dk = d;
  a.H = 1;
  a.nh[0] = N;
  a.per_head = N;
  a.ldo = N;
  a.sel_mask = sel_mask;
  a.sel_pre = sel_pre;
  a.sel_gates = sel_gates;
  a.aout = aout;
  a.words = words;
  a.ncols_out = ncols_out;
  a.hk = hk;
  a.act = act;
  const int64_t total = (int64_t)((ncols_out + LN - 1) / LN) * ((T + LM - 1) / LM);
  const int64_t grid = ((total + 7) / 8) * 8;
  hipLaunchKernelGGL((score_bf16_large_kernel<false, false, true>), dim3((unsigned)grid),
                     dim3(512), 2 * LSTAGE, st, a);
  return hipGetLastError();
}

}  // namespace omnimoe
