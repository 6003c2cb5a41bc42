// The second product of Eq. 14 as one dense GEMM over all experts, for layers whose routed
// pairs are dense (one head, K a sizeable fraction of N): y = A V with A[t, e] = a_p for the
// task p of token t routed to expert e and zero elsewhere, i.e. Eq. 14 with all experts in a
// single group. A is built in bf16 (a_p rounded to nearest even), V is transposed once so that
// the expert dimension is contiguous, the product runs on the MFMA logit kernel split over the
// expert dimension, and the split partials are added in split order, so y is deterministic.
// In the layer (one head, routing from the selection kernel) the first product runs dense as
// well: h = X U^T over all experts on the same MFMA kernel, whose epilogue keeps only the
// selected cells, A[t, e] = g * act(h[t, e]) in bf16, from a per-token selection mask; the
// schedule, the per-task dot and the densify pass are then not needed.
// A token's slots normally name distinct experts (the router picks K distinct cells), so each
// A[t, e] is a single a_p; when a caller's idx repeats an expert within a token, that entry is
// the sum of the repeated slots' a_p in slot order, so the result stays deterministic.
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

constexpr int kDenseChunk = 16384;  // columns of A built at a time (32 KiB of LDS)
constexpr int kDenseSlots = 16;     // a token's slots held per thread (hk <= 4096)

// Row t of A: the token's K (expert, a) pairs are loaded once into registers; then, chunk by
// chunk of columns, the chunk is zeroed in LDS, the pairs that fall in it are placed, and it
// is written out with 16-byte stores. Placement first marks each column with the number of
// one slot that falls in it (any one: concurrent plain stores); a slot that then reads back
// another slot's number shares its expert with it. Without such a slot in the chunk (the
// router's case) every slot stores its own value. Otherwise the slot whose mark survived
// sums, in slot order, the a of every slot with its expert (read again from memory), so the
// result does not depend on which store won.
__global__ __launch_bounds__(256) void densify_kernel(const int32_t* __restrict__ idx,
                                                      const float* __restrict__ a,
                                                      uint16_t* __restrict__ A, int hk,
                                                      int64_t N, int64_t kpad) {
  __shared__ __attribute__((aligned(16))) uint16_t row[kDenseChunk];
  __shared__ __attribute__((aligned(16))) uint16_t mark[kDenseChunk];  // slot number + 1
  const int64_t t = blockIdx.x;
  const int tid = threadIdx.x;
  int e[kDenseSlots];
  uint16_t v[kDenseSlots];
  float av[kDenseSlots];
  // All 2 * kDenseSlots loads in flight at once: unconditional, a slot past hk reading the last
  // slot and masked afterwards (guarded loads would each wait for the previous one).
#pragma unroll
  for (int q = 0; q < kDenseSlots; ++q) {
    const int j = q * 256 + tid < hk ? q * 256 + tid : hk - 1;
    e[q] = idx[t * hk + j];
    av[q] = a[t * hk + j];
  }
#pragma unroll
  for (int q = 0; q < kDenseSlots; ++q) {
    const bool ok = q * 256 + tid < hk;
    e[q] = ok ? e[q] : -1;
    v[q] = ok ? bf16_rne(av[q]) : (uint16_t)0;
  }
  uint4* dst_row = (uint4*)(A + t * kpad);
  for (int64_t c0 = 0; c0 < kpad; c0 += kDenseChunk) {
    for (int i = tid; i < kDenseChunk / 8; i += 256) {
      ((uint4*)row)[i] = make_uint4(0, 0, 0, 0);
      ((uint4*)mark)[i] = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kDenseSlots; ++q) {
      const int64_t c = (int64_t)e[q] - c0;
      if (e[q] >= 0 && e[q] < N && c >= 0 && c < kDenseChunk) mark[c] = (uint16_t)(q * 256 + tid + 1);
    }
    __syncthreads();
    int shared_expert = 0;
#pragma unroll
    for (int q = 0; q < kDenseSlots; ++q) {
      const int64_t c = (int64_t)e[q] - c0;
      if (e[q] >= 0 && e[q] < N && c >= 0 && c < kDenseChunk)
        shared_expert |= mark[c] != (uint16_t)(q * 256 + tid + 1);
    }
    if (!__syncthreads_or(shared_expert)) {
#pragma unroll
      for (int q = 0; q < kDenseSlots; ++q) {
        const int64_t c = (int64_t)e[q] - c0;
        if (e[q] >= 0 && e[q] < N && c >= 0 && c < kDenseChunk) row[c] = v[q];
      }
    } else {
      for (int q = 0; q < kDenseSlots; ++q) {
        const int64_t c = (int64_t)e[q] - c0;
        if (e[q] >= 0 && e[q] < N && c >= 0 && c < kDenseChunk &&
            mark[c] == (uint16_t)(q * 256 + tid + 1)) {
          float sum = 0.f;
          for (int jj = 0; jj < hk; ++jj)
            if (idx[t * hk + jj] == e[q]) sum += a[t * hk + jj];
          row[c] = bf16_rne(sum);
        }
      }
    }
    __syncthreads();
    const int64_t n = kpad - c0 < kDenseChunk ? kpad - c0 : kDenseChunk;  // a multiple of 64
    for (int i = tid; i < n / 8; i += 256) {
      // non-temporal: A (T x N bf16) is far larger than the caches and read once by the GEMM
      typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
      const uint4 q = ((const uint4*)row)[i];
      const u32x4_t o = {q.x, q.y, q.z, q.w};
      __builtin_nontemporal_store(o, (u32x4_t*)&dst_row[c0 / 8 + i]);
    }
    __syncthreads();
  }
}

// Vt[c, e] = V[e, c] for e < N, zero for N <= e < kpad; 64 x 64 tiles through LDS, 16-byte
// loads (eight d values of one expert) and 16-byte stores (eight experts of one d index).
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ V,
                                                             uint16_t* __restrict__ Vt,
                                                             int64_t N, int d, int64_t kpad) {
  __shared__ uint16_t tile[64][72];  // [expert][d index], rows padded to 144 bytes
  const int64_t e0 = (int64_t)blockIdx.x * 64;
  const int c0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int i = q * 256 + tid;  // 512 chunks: expert i / 8, d indices 8 (i % 8) .. + 7
    const int r = i >> 3, k = (i & 7) * 8;
    const int64_t e = e0 + r;
    uint4 x = make_uint4(0, 0, 0, 0);
    if (e < N) x = *(const uint4*)(V + e * d + c0 + k);
    *(uint4*)&tile[r][k] = x;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int i = q * 256 + tid;  // 512 chunks: d index i / 8, experts 8 (i % 8) .. + 7
    const int c = i >> 3, k = (i & 7) * 8;
    uint16_t w[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) w[m] = tile[k + m][c];
    const uint4 o = make_uint4((uint32_t)w[0] | ((uint32_t)w[1] << 16),
                               (uint32_t)w[2] | ((uint32_t)w[3] << 16),
                               (uint32_t)w[4] | ((uint32_t)w[5] << 16),
                               (uint32_t)w[6] | ((uint32_t)w[7] << 16));
    if (e0 + k < kpad) *(uint4*)(Vt + (int64_t)(c0 + c) * kpad + e0 + k) = o;
  }
}

// y[i] = sum over splits z = 0, 1, ... of part[z][i], four elements per thread.
__global__ __launch_bounds__(256) void reduce_splits_kernel(const float* __restrict__ part,
                                                            float* __restrict__ y, int64_t n4,
                                                            int splits, int64_t stride4) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * 256) {
    float4 s = ((const float4*)part)[i];
    for (int z = 1; z < splits; ++z) {
      const float4 p = ((const float4*)part)[z * stride4 + i];
      s.x += p.x;
      s.y += p.y;
      s.z += p.z;
      s.w += p.w;
    }
    ((float4*)y)[i] = s;
  }
}

// Selection of one token as a bitmask over expert ids (bit e % 32 of word e / 32), the number
// of selected experts in the words before each word, and the gates in expert-id order:
// gsorted[t, r] = gate of the selected expert of rank r. One workgroup per token; the mask and
// the prefix counts are built in LDS (bits set with LDS atomic ORs, which commute), sized per
// launch (words x 6 bytes: the counts fit in 16 bits, hk <= 4096) so that several tokens share a
// compute unit. The layer's ids come from the selection kernel and are distinct within a token.
constexpr int kMaskWordsMax = 9216;  // words of one token (N up to 294912 experts)

size_t select_mask_lds_bytes(int words) { return (size_t)words * 6 + 16; }

__global__ __launch_bounds__(256) void select_mask_kernel(const int32_t* __restrict__ idx,
                                                          const float* __restrict__ gates,
                                                          uint32_t* __restrict__ mask,
                                                          int32_t* __restrict__ pre,
                                                          float* __restrict__ gsorted, int hk,
                                                          int64_t N, int words) {
  extern __shared__ __attribute__((aligned(16))) unsigned char sm[];
  uint32_t* lm = (uint32_t*)sm;                 // [words]
  uint16_t* lpre = (uint16_t*)(sm + words * 4);  // [words]
  __shared__ int wtot[4];
  const int64_t t = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // the token's slots, kDenseSlots per thread, all loads in flight at once (a slot past hk reads
  // the last slot and is dropped)
  int e[kDenseSlots];
  float gv[kDenseSlots];
#pragma unroll
  for (int q = 0; q < kDenseSlots; ++q) {
    const int j = q * 256 + tid < hk ? q * 256 + tid : hk - 1;
    e[q] = idx[t * hk + j];
    gv[q] = gates[t * hk + j];
  }
  for (int w = tid; w < words; w += 256) lm[w] = 0u;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kDenseSlots; ++q) {
    if (q * 256 + tid >= hk || e[q] < 0 || e[q] >= N) e[q] = -1;
    if (e[q] >= 0) atomicOr(&lm[e[q] >> 5], 1u << (e[q] & 31));
  }
  __syncthreads();
  // exclusive prefix of the words' popcounts: thread tid sums a contiguous run of words, the run
  // sums are scanned within each wave and then across the four waves, and each run is walked again
  const int per = (words + 255) / 256;
  const int w_lo = tid * per < words ? tid * per : words;
  const int w_hi = w_lo + per < words ? w_lo + per : words;
  int run = 0;
  for (int w = w_lo; w < w_hi; ++w) run += __popc(lm[w]);
  const int excl = wave_excl_scan_i32(run);
  if (lane == kWave - 1) wtot[wv] = excl + run;
  __syncthreads();
  int c = excl;
  for (int v = 0; v < wv; ++v) c += wtot[v];
  for (int w = w_lo; w < w_hi; ++w) {
    lpre[w] = (uint16_t)c;
    c += __popc(lm[w]);
  }
  __syncthreads();
  for (int w = tid; w < words; w += 256) {
    mask[t * words + w] = lm[w];
    pre[t * words + w] = lpre[w];
  }
#pragma unroll
  for (int q = 0; q < kDenseSlots; ++q) {
    if (e[q] >= 0) {
      const int w = e[q] >> 5;
      const int r = lpre[w] + __popc(lm[w] & ((1u << (e[q] & 31)) - 1u));
      gsorted[t * hk + r] = gv[q];
    }
  }
}

struct DensePlan {
  int splits;
  int kchunk;
  int64_t kpad;
};

DensePlan dense_plan(const Shape& s) {
  const int64_t tiles = ((s.T + 255) / 256) * (((int64_t)s.d + 255) / 256);
  int64_t splits = (512 + tiles - 1) / tiles;
  const int64_t max_splits = (s.N + 511) / 512;  // at least eight 64-wide k steps per split
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  DensePlan p;
  p.splits = (int)splits;
  p.kchunk = (int)(((s.N + splits * 64 - 1) / (splits * 64)) * 64);
  p.kpad = (int64_t)p.kchunk * splits;
  return p;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

bool dense_accumulate(const Shape& s) {
  return s.bf16 && s.H == 1 && s.d % 64 == 0 && s.hk <= 256 * kDenseSlots &&
         (int64_t)s.K * kDenseRatio >= s.N && (double)s.T * (double)s.N * 2.0 <= kDenseMaxBytes;
}

size_t dense_accumulate_ws_bytes(const Shape& s) {
  if (!dense_accumulate(s)) return 0;
  const DensePlan p = dense_plan(s);
  size_t b = align256((size_t)s.T * p.kpad * 2);              // A
  b += align256((size_t)s.d * p.kpad * 2);                    // V transposed
  if (p.splits > 1) b += align256((size_t)p.splits * s.T * s.d * 4);  // split partials
  return b;
}

namespace {

// y = A V from A [T, kpad] bf16 at the start of ws (V transposed, split-K product, partials
// added in split order).
hipError_t launch_dense_product(const Shape& s, const void* v, float* y, void* ws,
                                hipStream_t st) {
  const DensePlan p = dense_plan(s);
  char* w = (char*)ws;
  uint16_t* A = (uint16_t*)w;
  w += align256((size_t)s.T * p.kpad * 2);
  uint16_t* Vt = (uint16_t*)w;
  w += align256((size_t)s.d * p.kpad * 2);
  float* part = p.splits > 1 ? (float*)w : y;
  hipLaunchKernelGGL(transpose_bf16_kernel, dim3((unsigned)(p.kpad / 64), (unsigned)(s.d / 64)),
                     dim3(256), 0, st, (const uint16_t*)v, Vt, s.N, s.d, p.kpad);
  hipError_t e = launch_gemm_splitk(s.T, s.d, A, p.kpad, Vt, p.kpad, p.kchunk, p.splits, part, st);
  if (e != hipSuccess) return e;
  if (p.splits > 1) {
    const int64_t n4 = s.T * (int64_t)s.d / 4;
    int64_t blocks = (n4 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(reduce_splits_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                       (const float*)part, y, n4, p.splits, n4);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dense_accumulate(const Shape& s, const void* v, const int32_t* idx,
                                   const float* abuf, float* y, void* ws, hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const DensePlan p = dense_plan(s);
  hipLaunchKernelGGL(densify_kernel, dim3((unsigned)s.T), dim3(256), 0, st, idx, abuf,
                     (uint16_t*)ws, s.hk, s.N, p.kpad);
  return launch_dense_product(s, v, y, ws, st);
}

bool dense_dot(const Shape& s) {
  return dense_accumulate(s) && s.B == 1 && dense_plan(s).kpad / 32 <= kMaskWordsMax;
}

size_t dense_dot_ws_bytes(const Shape& s) {
  if (!dense_dot(s)) return 0;
  const int64_t words = dense_plan(s).kpad / 32;
  return dense_accumulate_ws_bytes(s) + 2 * align256((size_t)s.T * words * 4) +
         align256((size_t)s.T * s.hk * 4);
}

namespace {

struct MaskBufs {
  uint32_t* mask;
  int32_t* pre;
  float* gsorted;
  int64_t words;
};

MaskBufs mask_bufs(const Shape& s, void* ws) {
  MaskBufs b;
  b.words = dense_plan(s).kpad / 32;
  char* w = (char*)ws + dense_accumulate_ws_bytes(s);
  b.mask = (uint32_t*)w;
  w += align256((size_t)s.T * b.words * 4);
  b.pre = (int32_t*)w;
  w += align256((size_t)s.T * b.words * 4);
  b.gsorted = (float*)w;
  return b;
}

}  // namespace

hipError_t launch_select_mask(const Shape& s, const int32_t* idx, const float* gates, void* ws,
                              hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const MaskBufs b = mask_bufs(s, ws);
  hipLaunchKernelGGL(select_mask_kernel, dim3((unsigned)s.T), dim3(256),
                     select_mask_lds_bytes((int)b.words), st, idx, gates, b.mask, b.pre, b.gsorted,
                     s.hk, s.N, (int)b.words);
  return hipGetLastError();
}

hipError_t launch_dense_dot(const Shape& s, const void* x, const void* u, void* ws,
                            hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  const MaskBufs b = mask_bufs(s, ws);
  return launch_gemm_act_mask(s.T, (int)s.N, (int)dense_plan(s).kpad, x, s.d, u, b.mask, b.pre,
                              b.words, b.gsorted, s.hk, s.act, (uint16_t*)ws, st);
}

hipError_t launch_dense_routed_sum(const Shape& s, const void* v, float* y, void* ws,
                                   hipStream_t st) {
  if (s.T == 0) return hipSuccess;
  return launch_dense_product(s, v, y, ws, st);
}

}  // namespace omnimoe
