// HIP kernels for gfx950 (MI355X): one step of batched beam decoding with LMBR
// n-gram posteriors (Algorithm 1 with sentence batching, Eq. 1 and Eq. 2 of
// Iglesias et al., NAACL-HLT 2018).
//
// Per step, for B sentences x K beams (M = B*K rows):
//   k_gemm        logits[M, V] = hidden[M, H] . W[V, H]^T + bias     (bf16 MFMA, fp32 acc)
//   k_score       per (sentence, V-tile): log-softmax partials (max, sum exp),
//                 the LMBR term added from the sparse tables, and each row's
//                 partial top-K of logit + lambda * L
//   k_merge       per sentence: exact top-K over the K x K-candidate lists with
//                 the running scores (TopB), EOS push/mask, realignment of the
//                 histories by backpointer, and the next step's context probes
//   k_traceback   GetBestHypothesis over F at the end of decoding
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "kernels.h"

namespace lmbr {
namespace dev {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Irwin-Hall sum of 12 uniforms of 20 bits from mix64(h + r), r = 0..3,
// centred and scaled by 2^-20: exact in fp32.
__device__ __forceinline__ float irwin_hall(uint64_t h) {
  int32_t s = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint64_t w = mix64(h + (uint64_t)r);
    s += (int32_t)(w & 0xFFFFFu) + (int32_t)((w >> 20) & 0xFFFFFu) + (int32_t)((w >> 40) & 0xFFFFFu);
  }
  s -= 6 * ((1 << 20) - 1);
  return (float)s * 0x1p-20f;
}

__device__ __forceinline__ uint16_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Raise device fault bits (LMBR_DEV_*); a null flag (no context) ignores them.
__device__ __forceinline__ void flag_fault(int *err, int bits) {
  if (err) atomicOr(err, bits);
}

// Linear-probing lookup of a packed history; returns (offset, count) or (0, 0).
// A full pass without an empty slot (a corrupt table) raises LMBR_DEV_TABLE.
__device__ __forceinline__ int2 probe(const SentTable &tb, uint64_t key, int *err) {
  uint32_t h = (uint32_t)(mix64(key) & tb.mask);
  for (uint32_t step = 0; step <= tb.mask; ++step) {
    const Slot sl = tb.slots[h];
    if (sl.key == key) return make_int2((int)sl.off, (int)sl.cnt);
    if (sl.key == kEmptyKeyDev) return make_int2(0, 0);
    h = (h + 1) & tb.mask;
  }
  flag_fault(err, LMBR_DEV_TABLE);
  return make_int2(0, 0);
}

// The slot of a packed history, or -1 (same probe sequence).
__device__ __forceinline__ int probe_slot(const SentTable &tb, uint64_t key, int *err) {
  uint32_t h = (uint32_t)(mix64(key) & tb.mask);
  for (uint32_t step = 0; step <= tb.mask; ++step) {
    const uint64_t k = tb.slots[h].key;
    if (k == key) return (int)h;
    if (k == kEmptyKeyDev) return -1;
    h = (h + 1) & tb.mask;
  }
  flag_fault(err, LMBR_DEV_TABLE);
  return -1;
}

// Dense layout: the row of L for a slot whose last words are ctx (len words
// of history): the longest suffix of at most three words that is a history
// of the table (longer contexts have no n-grams), row 0 when none is.
__device__ __forceinline__ int dense_row(const SentTable &tb, uint64_t ctx, int len, int *err) {
  for (int w = min(len, 3); w >= 1; --w) {
    const int h = probe_slot(tb, ctx & ((1ull << (21 * w)) - 1), err);
    if (h >= 0) return (int)tb.slot_row[h];
  }
  return 0;
}

// (x desc, v asc): "a ranks before b"
__device__ __forceinline__ bool better(float ax, int av, float bx, int bv) {
  return ax > bx || (ax == bx && av < bv);
}
__device__ __forceinline__ bool better_d(double ax, int av, double bx, int bv) {
  return ax > bx || (ax == bx && av < bv);
}

// Cross-lane moves without LDS: DPP within rows of 16 lanes, then readlane
// across the four rows of a wave64.  Encodings (GFX9 DPP16): quad_perm
// [1,0,3,2] = 0xB1, quad_perm [2,3,0,1] = 0x4E, row_half_mirror = 0x141
// (lane i <-> 7-i within 8), row_mirror = 0x140 (lane i <-> 15-i).
constexpr int kDppXor1 = 0xB1;
constexpr int kDppXor2 = 0x4E;
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;
constexpr int kDppShr1 = 0x111;      // row_shr:1 (lane i takes lane i - 1 within its row)

template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(dpp_i<CTRL>(__float_as_int(x)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double x) {
  const long long b = __double_as_longlong(x);
  const int lo = dpp_i<CTRL>((int)(b & 0xFFFFFFFFll)), hi = dpp_i<CTRL>((int)(b >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
__device__ __forceinline__ float rdlane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}
__device__ __forceinline__ int rdlane_i(int x, int l) { return __builtin_amdgcn_readlane(x, l); }
__device__ __forceinline__ double rdlane_d(double x, int l) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)(b & 0xFFFFFFFFll), l);
  const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, dpp_f<kDppXor1>(x));
  x = fmaxf(x, dpp_f<kDppXor2>(x));
  x = fmaxf(x, dpp_f<kDppHalfMirror>(x));
  return fmaxf(x, dpp_f<kDppMirror>(x));
}
__device__ __forceinline__ float wave_max(float x) {
  x = row16_max(x);
  return fmaxf(fmaxf(rdlane_f(x, 0), rdlane_f(x, 16)), fmaxf(rdlane_f(x, 32), rdlane_f(x, 48)));
}
__device__ __forceinline__ float wave_min(float x) {
  x = fminf(x, dpp_f<kDppXor1>(x));
  x = fminf(x, dpp_f<kDppXor2>(x));
  x = fminf(x, dpp_f<kDppHalfMirror>(x));
  x = fminf(x, dpp_f<kDppMirror>(x));
  return fminf(fminf(rdlane_f(x, 0), rdlane_f(x, 16)), fminf(rdlane_f(x, 32), rdlane_f(x, 48)));
}
__device__ __forceinline__ float wave_sum(float x) {
  x += dpp_f<kDppXor1>(x);
  x += dpp_f<kDppXor2>(x);
  x += dpp_f<kDppHalfMirror>(x);
  x += dpp_f<kDppMirror>(x);
  return (rdlane_f(x, 0) + rdlane_f(x, 16)) + (rdlane_f(x, 32) + rdlane_f(x, 48));
}

template <int CTRL>
__device__ __forceinline__ void argmax_step(float &x, int &v) {
  const float ox = dpp_f<CTRL>(x);
  const int ov = dpp_i<CTRL>(v);
  if (better(ox, ov, x, v)) { x = ox; v = ov; }
}
// Wave-wide best (x, v); every lane receives it.
__device__ __forceinline__ void wave_argmax(float &x, int &v) {
  argmax_step<kDppXor1>(x, v);
  argmax_step<kDppXor2>(x, v);
  argmax_step<kDppHalfMirror>(x, v);
  argmax_step<kDppMirror>(x, v);
  float bx = rdlane_f(x, 0);
  int bv = rdlane_i(v, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const float ox = rdlane_f(x, r);
    const int ov = rdlane_i(v, r);
    if (better(ox, ov, bx, bv)) { bx = ox; bv = ov; }
  }
  x = bx;
  v = bv;
}

template <int CTRL>
__device__ __forceinline__ void argmax_step_d(double &x, int &v) {
  const double ox = dpp_d<CTRL>(x);
  const int ov = dpp_i<CTRL>(v);
  if (better_d(ox, ov, x, v)) { x = ox; v = ov; }
}
__device__ __forceinline__ void wave_argmax_d(double &x, int &v) {
  argmax_step_d<kDppXor1>(x, v);
  argmax_step_d<kDppXor2>(x, v);
  argmax_step_d<kDppHalfMirror>(x, v);
  argmax_step_d<kDppMirror>(x, v);
  double bx = rdlane_d(x, 0);
  int bv = rdlane_i(v, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const double ox = rdlane_d(x, r);
    const int ov = rdlane_i(v, r);
    if (better_d(ox, ov, bx, bv)) { bx = ox; bv = ov; }
  }
  x = bx;
  v = bv;
}

// A lower bound on the K-th largest of the wave's elements, from G >= K
// disjoint lane groups (G a power of two <= 16): every group maximum is a
// distinct element, so the smallest of the G maxima is <= the K-th largest.
// `mx` is the lane's own maximum; -inf when a group holds no element.
__device__ __forceinline__ float group_bound(float mx, int G) {
  float g = mx;
  if (G <= 16) {
    g = fmaxf(g, dpp_f<kDppXor1>(g));
    g = fmaxf(g, dpp_f<kDppXor2>(g));
  }
  if (G <= 8) g = fmaxf(g, dpp_f<kDppHalfMirror>(g));
  if (G <= 4) g = fmaxf(g, dpp_f<kDppMirror>(g));
  if (G >= 4) return wave_min(g);
  const float r0 = rdlane_f(g, 0), r1 = rdlane_f(g, 16), r2 = rdlane_f(g, 32), r3 = rdlane_f(g, 48);
  if (G == 2) return fminf(fmaxf(r0, r1), fmaxf(r2, r3));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

}  // namespace dev

using namespace dev;

// ---------------------------------------------------------------------------
// Stand-in decoder state and beam-state bookkeeping
// ---------------------------------------------------------------------------
// Workgroup x covers row x / bpr, column block x % bpr: each thread makes
// eight consecutive columns of the row and writes them with one 16-byte store
// (H is a multiple of 64).
__global__ void k_synth_hidden(const uint64_t *__restrict__ hh, uint16_t *__restrict__ hidden,
                               int M, int H, int bpr) {
  const int m = (int)(blockIdx.x / (unsigned)bpr);
  const int c0 = 8 * ((int)(blockIdx.x % (unsigned)bpr) * (int)blockDim.x + (int)threadIdx.x);
  if (m >= M || c0 >= H) return;
  const uint64_t h = hh[m];
  uint32_t w[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t lo = bf16_rne(irwin_hall(mix64(h + (uint64_t)(c0 + 2 * k))));
    const uint32_t hi = bf16_rne(irwin_hall(mix64(h + (uint64_t)(c0 + 2 * k + 1))));
    w[k] = lo | (hi << 16);
  }
  *(uint4 *)(hidden + (size_t)m * H + c0) = make_uint4(w[0], w[1], w[2], w[3]);
}

__global__ void k_state_init(int B, int K, uint64_t seed, double *q, uint64_t *ctx, uint64_t *hh,
                             int *len, int *ranges, lmbr_sentence_record *sent) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * K) return;
  const int s = i / K, k = i % K;
  if (sent && k == 0) sent[s] = lmbr_sentence_record{-INFINITY, -INFINITY, 0, -1};
  q[i] = k == 0 ? 0.0 : -INFINITY;
  ctx[i] = 0;
  hh[i] = mix64(mix64(seed + 0x48ull) ^ (uint64_t)s);
  len[i] = 0;
#pragma unroll
  for (int r = 0; r < 6; ++r) ranges[i * 6 + r] = 0;
}

__global__ void k_state_probe(int B, int K, const SentTable *__restrict__ tabs,
                              const double *__restrict__ q, const uint64_t *__restrict__ ctx,
                              const int *__restrict__ len, int *__restrict__ ranges, int *err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * K * 3) return;
  const int row = i / 3, o = i % 3;          // order n = o + 2 needs n - 1 = o + 1 words
  const SentTable &tb = tabs[row / K];
  int2 r = make_int2(0, 0);
  if (tb.dense) {                             // dense layout: the row of L, in the first field
    if (o == 0 && q[row] != -INFINITY) r.x = dense_row(tb, ctx[row], len[row], err);
  } else if (q[row] != -INFINITY && len[row] >= o + 1) {
    const uint64_t key = ctx[row] & ((1ull << (21 * (o + 1))) - 1);
    r = probe(tb, key, err);
  }
  ranges[row * 6 + o * 2] = r.x;
  ranges[row * 6 + o * 2 + 1] = r.y;
}

__global__ void k_transpose_bf16(const uint16_t *__restrict__ src, uint16_t *__restrict__ dst,
                                 int rows, int cols) {
  // src [rows, cols] -> dst [cols, rows]
  __shared__ uint16_t tile[32][33];
  const int bx = blockIdx.x * 32, by = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 256 threads: 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int gr = by + r, gc = bx + tx;
    if (gr < rows && gc < cols) tile[r][tx] = src[(size_t)gr * cols + gc];
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int gr = bx + r, gc = by + tx;    // dst row = src col
    if (gr < cols && gc < rows) dst[(size_t)gr * rows + gc] = tile[tx][r];
  }
}

__global__ void k_gather_rows(uint32_t *__restrict__ dst, const uint32_t *__restrict__ src,
                              const int *__restrict__ rows, int n, int64_t words) {
  const int i = blockIdx.x;
  if (i >= n) return;
  const uint32_t *s = src + (int64_t)rows[i] * words;
  uint32_t *d = dst + (int64_t)i * words;
  for (int64_t w = threadIdx.x; w < words; w += blockDim.x) d[w] = s[w];
}

// x[i] += c (the constant lambda * theta0 of the dense layout of L, summed on
// the GPU after the upload).
__global__ void k_add_scalar(float *__restrict__ x, size_t n, float c) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    x[i] += c;
}

// ---------------------------------------------------------------------------
// Projection: bf16 MFMA GEMM, C[M, N] = A[M, Kd] . Bw[N, Kd]^T + bias
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Tile staging: NS stages of BK = 32 bf16 per row (four 16-byte chunks, 64
// bytes per row) for A (BM rows) and W (BN rows), filled straight from global
// memory by global_load_lds_dwordx4 (one instruction moves 16 rows x 64 bytes
// = 1 KB: lane i writes bytes 16i..16i+15, i.e. row i / 4, position i % 4).
// Chunk c of row r sits at position c ^ swz(r).  An MFMA operand read has 16
// consecutive lanes take one logical chunk of 16 consecutive rows; with 64 LDS
// banks (256 bytes = 4 rows per bank cycle) rows r, r+4, r+8, r+12 must use
// different positions, hence swz(r) = (r / 4) % 4.
__device__ __forceinline__ int lds_swz(int r) { return (r >> 2) & 3; }

// s_waitcnt with only the vector-memory counter bounded (expcnt and lgkmcnt
// left at their maxima): GFX9 encoding vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8]
// | vmcnt_hi[15:14].
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef __attribute__((address_space(3))) void *lds_ptr_t;

// The hot loop's phases are separated by sched_barrier(0): the compiler keeps
// the fragment reads where they are written (one k slice ahead of the MFMAs
// that consume them) and its wait-count pass emits the exact lgkmcnt for each
// MFMA group (LDS reads complete in order).  Without the fences it re-reads
// fragments with a full wait before every MFMA pair.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

template <int BM, int BN, int WM, int WN>
struct TileShape {
  static constexpr int WAVES_N = BN / WN;
  static constexpr int NW = (BM / WM) * WAVES_N;       // waves per workgroup
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int NF = TM + TN;                   // fragments per 16-wide k slice
  static constexpr int BK = 32;                        // bf16 per row per stage (two k slices)
  static constexpr int ROWB = BK * 2;                  // bytes per staged row
  static constexpr int NS = 4;                         // LDS stages
  static constexpr int STAGE = (BM + BN) * ROWB;       // bytes per stage
  static constexpr int CHUNKS = (BM + BN) / 16;        // 1 KB load instructions per stage
  static constexpr int LPW = CHUNKS / NW;              // ... per wave
  static constexpr int LDS_BYTES = NS * STAGE;
  static_assert(CHUNKS % NW == 0, "load chunks must split evenly over the waves");
  static_assert(NS == 4, "wait_stage covers two later stages");
};

// Workgroup barrier without a memory wait: on this target s_barrier does not
// wait for the wave's outstanding memory operations.  Safe in the main loop,
// where every LDS read before it has been consumed and the stage loads are
// awaited with explicit vmcnt waits.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
// Barrier that publishes the wave's LDS writes first (lgkmcnt(0), other
// counters at their maxima).
__device__ __forceinline__ void lds_sync_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One BM x BN output tile: acc = A[m0 : m0 + BM, :] . Bw[n0 : n0 + BN, :]^T,
// with rows past M and N clamped to the last row (their results are not
// used); with amap (LDS, BM entries) A's rows are amap[0 .. BM) instead.  On entry the LDS stage buffers (at byte address lds0) must be free
// in every wave of the workgroup; on return every wave has finished its own
// reads of them but other waves may still be reading (a barrier is needed
// before the buffers are written again).
template <int BM, int BN, int WM, int WN>
__device__ __forceinline__ void mma_tile(const uint16_t *__restrict__ A, const uint16_t *__restrict__ Bw, int M,
                                         int N, int Kd, int m0, int n0, uint32_t lds0, int wid, int lane,
                                         f32x16_t (&acc)[WM / 32][WN / 32], const int *amap = nullptr) {
  using S = TileShape<BM, BN, WM, WN>;
  constexpr int TM = S::TM, TN = S::TN, NF = S::NF, BK = S::BK, ROWB = S::ROWB, NS = S::NS;
  constexpr int STAGE = S::STAGE, LPW = S::LPW;
  // Opaque copies: when this loop runs once per tile of a longer kernel, the
  // per-lane set-up below is recomputed per call instead of being hoisted and
  // kept live (in registers) through the caller's epilogue.
  asm volatile("" : "+v"(lane), "+s"(wid), "+s"(Kd), "+s"(M), "+s"(N), "+s"(lds0));
  const int wm = wid / S::WAVES_N, wn = wid % S::WAVES_N;

  // this lane's global source for each of the wave's load instructions
  const uint16_t *src[LPW];
  int dst_off[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int q = wid * LPW + j;                 // 1 KB chunk of the stage
    const int rr = q * 16 + (lane >> 2);         // staged row (A rows first, then W rows)
    const int pos = lane & 3;
    const int c = pos ^ lds_swz(rr < BM ? rr : rr - BM);
    if (rr < BM) src[j] = A + (size_t)(amap ? amap[rr] : min(m0 + rr, M - 1)) * Kd + c * 8;
    else src[j] = Bw + (size_t)min(n0 + rr - BM, N - 1) * Kd + c * 8;
    dst_off[j] = q * 1024;
  }
  // The direct-to-LDS loads are issued as inline asm: the compiler models them
  // as counting on LGKM as well, which would force every LDS fragment wait in
  // the loop to lgkmcnt(0).  Their completion is awaited explicitly with the
  // vmcnt waits below, before the barrier that publishes each stage.
  auto issue = [&](int kt) {
    const uint32_t base = lds0 + (uint32_t)((kt % NS) * STAGE);
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src[j] + kt * BK), "{m0}"(base + dst_off[j])
                   : "memory");
  };

  // LDS byte offsets of this lane's fragments within a stage, per k slice
  uint32_t foff[2][NF];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int chunk = kk * 2 + (lane >> 5);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WM + i * 32 + (lane & 31);
      foff[kk][i] = lds0 + r * ROWB + ((chunk ^ lds_swz(r)) << 4);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int r = wn * WN + j * 32 + (lane & 31);
      foff[kk][TM + j] = lds0 + BM * ROWB + r * ROWB + ((chunk ^ lds_swz(r)) << 4);
    }
  }
  // fragments are carried as 32-bit words (bf16 vectors carried across the
  // loop's branches get split into halves and re-packed by the compiler)
  u32x4_t fa[NF], fb[NF];                       // slice 0 and slice 1 of a stage
  auto read_frags = [&](u32x4_t (&f)[NF], int kt, int kk) {
    const uint32_t sb = (uint32_t)((kt % NS) * STAGE);
#pragma unroll
    for (int i = 0; i < NF; ++i)
      f[i] = *(const __attribute__((address_space(3))) u32x4_t *)(uintptr_t)(foff[kk][i] + sb);
  };

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  auto mfmas = [&](const u32x4_t (&f)[NF]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, f[i]),
                                                            __builtin_bit_cast(bf16x8_t, f[TM + j]),
                                                            acc[i][j], 0, 0, 0);
      }
  };
  // wait until stage s has landed, given that stages s+1 .. s+later are in flight
  auto wait_stage = [&](int later) {
    if (later >= 2) wait_vmcnt<2 * LPW>();
    else if (later == 1) wait_vmcnt<LPW>();
    else wait_vmcnt<0>();
  };

  // Pipeline (one barrier per stage, between the stage's two k slices):
  //   stage j: read slice 1 of j | MFMA slice 0 of j | wait stage j+1, barrier,
  //            load stage j+NS-1 into stage j-1's buffer, read slice 0 of j+1 |
  //            MFMA slice 1 of j
  const int nk = Kd / BK;
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < nk) issue(p);
  wait_stage(min(nk - 1, NS - 2));
  lds_barrier();
  read_frags(fa, 0, 0);
  for (int kt = 0; kt + 1 < nk; ++kt) {
    sched_fence();
    read_frags(fb, kt, 1);
    sched_fence();
    mfmas(fa);
    sched_fence();
    wait_stage(max(0, min(nk - kt - 2, NS - 3)));
    lds_barrier();
    if (kt + NS - 1 < nk) issue(kt + NS - 1);
    read_frags(fa, kt + 1, 0);
    sched_fence();
    mfmas(fb);
  }
  // the last stage, peeled so that the loop body's waits stay exact
  sched_fence();
  read_frags(fb, nk - 1, 1);
  sched_fence();
  mfmas(fa);
  sched_fence();
  mfmas(fb);
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
void k_gemm(const uint16_t *__restrict__ A, const uint16_t *__restrict__ Bw,
            const float *__restrict__ bias, float *__restrict__ C, int M, int N, int Kd,
            int64_t ldc, int nMb, int nNb, int NT, int remap, const double *__restrict__ q,
            int *__restrict__ live_count) {
  using S = TileShape<BM, BN, WM, WN>;
  constexpr int TM = S::TM, TN = S::TN;
  constexpr int NTH = S::NW * 64;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[S::LDS_BYTES];
  __shared__ __attribute__((aligned(16))) int s_map[BM];
  __shared__ int s_wsum[S::NW];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  int bid = blockIdx.x;
  const int nstrips = (nNb + NT - 1) / NT;
  if (remap) {
    // Consecutive workgroups land on different XCDs; give each XCD a contiguous
    // run of strips so the M-blocks sharing a W block share that XCD's L2.
    const int per = (nMb * nstrips) >> 3;
    bid = (bid & 7) * per + (bid >> 3);
  }
  // workgroup = one M-block x one strip of NT column tiles, taken in order
  // (the block's rows stay in L2 across its strip)
  int mb = bid % nMb, strip = bid / nMb, nt_strip = NT;
  int m0 = mb * BM;
  const int wm = wid / S::WAVES_N, wn = wid % S::WAVES_N;

  // With running scores q, only the live rows (finite score) are projected:
  // the workgroup lists the beam's live rows in row order (a ballot and a
  // cross-wave prefix count per NTH rows), block mb takes live rows m0 ..
  // m0 + BM - 1 and writes each to its own row of C.  Rows past the last live
  // one repeat it (a valid row for the operand loads) and are not stored.
  // When fewer blocks are live than the grid was cut for (the first step of a
  // decode, or a batch whose sentences have finished), the live blocks take
  // shorter strips, as many as spread their tiles over the whole grid, and
  // the rows are listed again for the block this workgroup then takes.
  int mrows = M - m0;                                  // rows of this block that are stored
  const bool use_map = q != nullptr;
  if (use_map) {
    auto list_rows = [&]() {
      int n = 0;
      for (int c0 = 0; c0 < M; c0 += NTH) {
        const int r = c0 + tid;
        const bool lv = r < M && q[r] != -INFINITY;
        const uint64_t bal = __ballot(lv);
        const int wpre =
            __builtin_amdgcn_mbcnt_hi((unsigned)(bal >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)bal, 0u));
        if (lane == 0) s_wsum[wid] = __popcll(bal);
        __syncthreads();
        int before = n, total = n;
#pragma unroll
        for (int w = 0; w < S::NW; ++w) {
          before += w < wid ? s_wsum[w] : 0;
          total += s_wsum[w];
        }
        const int p = before + wpre;
        if (lv && p >= m0 && p < m0 + BM) s_map[p - m0] = r;
        n = total;
        __syncthreads();                               // s_wsum is rewritten by the next chunk
      }
      return n;
    };
    const int n = list_rows();
    if (blockIdx.x == 0 && tid == 0 && live_count) *live_count = n;
    const int nlb = (n + BM - 1) / BM;                 // live blocks (uniform)
    if (nlb == 0) return;
    if (nlb < nMb) {
      int t = 1;
      while (nlb * ((nNb + t - 1) / t) > (int)gridDim.x) ++t;
      const int bw = blockIdx.x;
      if (bw >= nlb * ((nNb + t - 1) / t)) return;
      mb = bw % nlb;
      strip = bw / nlb;
      nt_strip = t;
      const int m0_first = m0;
      m0 = mb * BM;
      if (m0 != m0_first) list_rows();
    }
    if (m0 >= n) return;
    mrows = n - m0;
    for (int i = mrows + tid; i < BM; i += NTH) s_map[i] = s_map[mrows - 1];
    __syncthreads();
  }

  // Make the epilogue's kernel arguments resident now: a scalar load still in
  // flight inside the main loop would force every LDS wait there to lgkmcnt(0).
  asm volatile("" ::"s"(bias), "s"(C), "s"(ldc), "s"(mrows));
  const int nb_end = min(nNb, (strip + 1) * nt_strip);
  for (int nb = strip * nt_strip; nb < nb_end; ++nb) {
    const int n0 = nb * BN;
    f32x16_t acc[TM][TN];
    mma_tile<BM, BN, WM, WN>(A, Bw, M, N, Kd, m0, n0, (uint32_t)(uintptr_t)(lds_ptr_t)smem, wid, lane, acc,
                             use_map ? s_map : nullptr);
    // every wave's fragment reads are done: the next tile may refill the stages
    lds_barrier();

    // 32x32 accumulator layout: lane l holds column l % 32 and rows
    // 8 * (r / 4) + 4 * (l / 32) + r % 4 for r = 0..15.
    float bcol[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) bcol[j] = 0.f;
    if (bias) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn * WN + j * 32 + (lane & 31);
        bcol[j] = col < N ? bias[col] : 0.f;
      }
      // awaited here: a bias load still pending among the guarded stores below
      // makes the compiler wait for every earlier store before each later one
      wait_vmcnt<0>();
    }
    // non-temporal stores: the logits are consumed once by the score pass and
    // should not evict W from the last-level cache.  Four consecutive local
    // rows at a time (their C rows from the map, or m0 + local row), both of
    // the wave's column blocks of a row back to back: each row's 256 bytes
    // are written by two consecutive stores
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int lr = wm * WM + i * 32 + 8 * g + 4 * (lane >> 5);
        int rr[4];
        if (use_map) {
          const int4 rows = *(const int4 *)&s_map[lr];
          rr[0] = rows.x;
          rr[1] = rows.y;
          rr[2] = rows.z;
          rr[3] = rows.w;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) rr[u] = m0 + lr + u;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = n0 + wn * WN + j * 32 + (lane & 31);
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (lr + u < mrows && col < N)
              __builtin_nontemporal_store(acc[i][j][4 * g + u] + bcol[j], &C[(size_t)rr[u] * ldc + col]);
        }
      }
  }
}

// Order-preserving 64-bit keys: (x descending, word ascending) <=> key descending.
// Key 0 means "no entry" (below every real key).
__device__ __forceinline__ uint32_t ord_f(float f) {
  const uint32_t b = __float_as_uint(f);
  return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}
__device__ __forceinline__ float unord_f(uint32_t h) {
  return __uint_as_float((h & 0x80000000u) ? (h ^ 0x80000000u) : ~h);
}
__device__ __forceinline__ uint64_t cand_key(float x, int v) {
  return ((uint64_t)ord_f(x) << 32) | (uint64_t)(~(uint32_t)v);
}
__device__ __forceinline__ Cand key_cand(uint64_t k) {
  const uint32_t h = (uint32_t)(k >> 32);
  return h == 0 ? Cand{-INFINITY, -1} : Cand{unord_f(h), (int)~(uint32_t)k};
}

// ---------------------------------------------------------------------------
// Score pass over logits in memory: log-softmax partials + LMBR add + per-row
// partial top-K, per strip of columns
// ---------------------------------------------------------------------------
// Grid (strip of NT tiles of 1024 columns, sentence); 4 waves per workgroup,
// wave w owning rows w, w + 4, .. of the sentence (K <= 16).  A wave takes its
// live rows in turn and each row's tiles in order (the next item's logits are
// loaded while the current one is scored; nothing is shared between waves, so
// there is no workgroup barrier).  Per (row, tile):
//   1. the row's logits, EOS bias and -inf past V; running log-softmax
//      partials (max, sum exp) per lane over the strip;
//   2. x = logit + lambda L(h, .): the sentence's dense history-free row
//      lambda (theta0 + theta1 p1) read straight from its table (one copy per
//      sentence, shared by its rows through the caches), plus the order 2..4
//      successors of the row's histories that fall in the tile, scattered
//      into the wave's LDS delta tile (each order's sorted list is walked by
//      a cursor that moves with the tiles); words outside an allowed set -inf;
//   3. candidates: x at or above the row's running K-th value (exact, from
//      the previous tiles) and, while the row has fewer than K, above a group
//      bound of this tile; a tile where no lane holds such a value is done
//      after one ballot; otherwise each candidate is inserted in turn into the
//      running list, held in lanes 0 .. K-1 (a ballot gives its position, a
//      one-lane DPP shift makes room), with no LDS traffic.
// After a row's last tile its partials are reduced over the wave and its list
// written: the layout the merge reads.
constexpr int SC_WAVES = 4;
constexpr int SC_TV = 1024;         // columns per tile

// Table arrays are read through global-address-space pointers: loads through
// generic pointers (the table's fields) would be flat loads, which also count
// on the LDS counter and so tie every LDS wait to the prefetch in flight.
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef const __attribute__((address_space(1))) i32x2_t *g_int2_p;
typedef const __attribute__((address_space(1))) uint32_t *g_u32_p;
typedef const __attribute__((address_space(1))) f32x4_t *g_f32x4_p;

// Five waves per SIMD (at most 96 VGPRs): the loads of one item are in
// flight while the other waves score theirs.
__global__ __launch_bounds__(SC_WAVES * 64) __attribute__((amdgpu_waves_per_eu(5)))
void k_score(const float *__restrict__ logits, int64_t ld, int V, int K, int ntiles, int NT, int nstrips, int G,
             const double *__restrict__ q, const int *__restrict__ ranges,
             const SentTable *__restrict__ tabs, const float *__restrict__ eos_bias, int eos,
             float lth2, float lth3, float lth4, const uint32_t *__restrict__ allowed, float *__restrict__ eosx,
             float2 *__restrict__ stats, Cand *__restrict__ topk, int *err) {
  constexpr int NG = SC_TV / 256;       // float4 groups per lane (16 values)
  __shared__ __attribute__((aligned(16))) float Dsh[SC_WAVES][SC_TV];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int strip = blockIdx.x, s = blockIdx.y;
  const int t0 = strip * NT, nt = min(NT, ntiles - t0);
  float *D = Dsh[wid];
  const SentTable tb = tabs[s];
  const g_int2_p ent = (g_int2_p)tb.entries;
  const g_f32x4_p udn0 = (g_f32x4_p)tb.uni_dense;
  const bool dense = tb.dense != nullptr;      // dense layout: each row reads its own row of L
  const int nrow = (K - wid + SC_WAVES - 1) / SC_WAVES;   // rows of this wave (uniform)
  const float lthn[3] = {lth2, lth3, lth4};
  const float bias_e = eos_bias ? eos_bias[s] : 0.f;
  const int Vpad = ((V + 255) >> 8) << 8;          // the dense row covers whole 256-column tiles
  const int Dt = (((V + 255) >> 8) + 2) >> 1;

#pragma unroll
  for (int g = 0; g < NG; ++g) *(float4 *)(&D[256 * g + 4 * lane]) = make_float4(0.f, 0.f, 0.f, 0.f);

  // live rows of the wave (bit i: row i); dead rows get empty partials
  unsigned live_mask = 0;
  for (int i = 0; i < nrow; ++i) {
    const int row = s * K + wid + SC_WAVES * i;
    if (q[row] != -INFINITY) {
      live_mask |= 1u << i;
    } else {
      const size_t o = (size_t)row * nstrips + strip;
      if (lane == 0) stats[o] = make_float2(-INFINITY, 0.f);
      if (lane < K) topk[o * K + lane] = Cand{-INFINITY, -1};
    }
  }
  if (live_mask == 0) return;

  // logits of (tile jt, row i) and the tile's dense history-free row into
  // nv / nl; the next item is loaded while the current one is scored
  float nv[4 * NG];
  float4 nl[NG];
  auto issue = [&](int jt, int i) {
    const int row = s * K + wid + SC_WAVES * i;
    int vb = (t0 + jt) * SC_TV, Vr = V;
    asm volatile("" : "+s"(vb), "+s"(Vr));   // no hoisted per-element masks
    const float *rp = logits + (size_t)row * ld;
    const g_f32x4_p udn = dense ? (g_f32x4_p)(tb.dense + (size_t)ranges[row * 6] * Vpad) : udn0;
    if (vb + SC_TV <= Vr) {                   // a whole tile (and Vpad >= V)
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const f32x4_t f = __builtin_nontemporal_load((const f32x4_t *)(rp + vb + 256 * g + 4 * lane));
        nv[4 * g] = f[0];
        nv[4 * g + 1] = f[1];
        nv[4 * g + 2] = f[2];
        nv[4 * g + 3] = f[3];
        const f32x4_t d = udn[(vb >> 2) + 64 * g + lane];
        nl[g] = make_float4(d[0], d[1], d[2], d[3]);
      }
    } else {                                  // the last tile: columns >= V are -inf
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int c = vb + 256 * g + 4 * lane;
        float4 f = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        if (c < Vr) f = *(const float4 *)(rp + c);
        nv[4 * g] = f.x;
        nv[4 * g + 1] = (c + 1 < Vr) ? f.y : -INFINITY;
        nv[4 * g + 2] = (c + 2 < Vr) ? f.z : -INFINITY;
        nv[4 * g + 3] = (c + 3 < Vr) ? f.w : -INFINITY;
        f32x4_t d = {0.f, 0.f, 0.f, 0.f};
        if (c < Vpad) d = udn[c >> 2];
        nl[g] = make_float4(d[0], d[1], d[2], d[3]);
      }
    }
  };
  auto next_live = [&](int i) {
    do ++i;
    while (i < nrow && !((live_mask >> i) & 1u));
    return i;
  };

  // state of the current row: per order 2..4 a cursor into its sorted
  // successor list, the list's end and the word at the cursor (INT_MAX: none);
  // running log-softmax partials of the lane's columns; running list (lane
  // k < K holds entry k) and its K-th value
  int cur[3], end[3], nxw[3];
  float mr = -INFINITY, sr = 0.f, tr = -INFINITY, rx = -INFINITY;
  int rv = -1;

  int cj = 0, ci = next_live(-1);
  issue(cj, ci);
  while (ci < nrow) {
    const int jt = cj, ii = ci;
    float val[4 * NG];
    float4 lw[NG];
#pragma unroll
    for (int e = 0; e < 4 * NG; ++e) val[e] = nv[e];
#pragma unroll
    for (int g = 0; g < NG; ++g) lw[g] = nl[g];
    if (++cj >= nt) {
      cj = 0;
      ci = next_live(ci);
    }
    if (ci < nrow) issue(cj, ci);

    const int row = s * K + wid + SC_WAVES * ii;
    if (jt == 0) {
      // a new row: first entry at or past the strip's first column of each
      // order's list, from the list's directory (first entry of each
      // 256-column tile) when it has one, else by counting the short list's
      // words below it
      mr = -INFINITY;
      sr = 0.f;
      tr = -INFINITY;
      rx = -INFINITY;
      rv = -1;
#pragma unroll
      for (int o = 0; o < 3; ++o) {
        cur[o] = end[o] = 0;
        nxw[o] = 0x7FFFFFFF;
        if (dense) continue;                  // the row of L holds every order
        const int off = ranges[row * 6 + 2 * o], cnt = ranges[row * 6 + 2 * o + 1];
        if (cnt == 0) continue;
        if (!(off >= 0 && cnt > 0 && (int64_t)off + cnt <= (int64_t)tb.n_entries)) {
          if (lane == 0) flag_fault(err, LMBR_DEV_TABLE);
          continue;
        }
        int c0;
        if (cnt > LMBR_DIR_MIN && off >= Dt) {
          const g_u32_p dir = (g_u32_p)(ent + off - Dt);
          c0 = (int)min(max(dir[t0 * (SC_TV / 256)], (uint32_t)off), (uint32_t)(off + cnt));
        } else {
          const bool below = lane < cnt && ent[off + lane].x < t0 * SC_TV;
          c0 = off + __popcll(__ballot(below));
        }
        cur[o] = c0;
        end[o] = off + cnt;
        nxw[o] = c0 < off + cnt ? ent[c0].x : 0x7FFFFFFF;
      }
    }

    const int v0 = (t0 + jt) * SC_TV;
    int vb = v0, Vr = V;
    asm volatile("" : "+s"(vb), "+s"(Vr));
    auto colv = [&](int e) { return vb + 256 * (e >> 2) + 4 * lane + (e & 3); };

    // 1. EOS bias; running log-softmax partials of the logits
    if (eos >= vb && eos < vb + SC_TV) {
#pragma unroll
      for (int e = 0; e < 4 * NG; ++e)
        if (colv(e) == eos) val[e] += bias_e;
    }
    {
      float m4[4] = {val[0], val[1], val[2], val[3]};
#pragma unroll
      for (int e = 4; e < 4 * NG; ++e) m4[e & 3] = fmaxf(m4[e & 3], val[e]);
      const float mx = fmaxf(mr, fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3])));
      if (mx != -INFINITY) {
        constexpr float kL2E = 1.44269504088896341f;
        const float nm = -mx * kL2E;
        float sa[4] = {mr == -INFINITY ? 0.f : sr * __builtin_amdgcn_exp2f(fmaf(mr, kL2E, nm)), 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4 * NG; ++e) sa[e & 3] += __builtin_amdgcn_exp2f(fmaf(val[e], kL2E, nm));
        sr = (sa[0] + sa[1]) + (sa[2] + sa[3]);
        mr = mx;
      }
    }

    // 2. order 2..4 successors in this tile into the delta tile: a walk from
    //    the cursor, only when the word there falls in the tile
    bool found = false;
#pragma unroll
    for (int o = 0; o < 3; ++o) {
      if (nxw[o] < vb + SC_TV) {
        int c = cur[o];
        const int e1 = end[o];
        int w;
        while (true) {
          const int e = c + lane;
          i32x2_t en = {0x7FFFFFFF, 0};
          if (e < e1) en = ent[e];
          const bool in = en.x < vb + SC_TV;
          if (in && en.x >= vb) D[en.x - vb] += lthn[o] * __int_as_float(en.y);
          const int nin = __popcll(__ballot(in));
          c += nin;
          if (nin < 64) {
            w = __shfl(en.x, nin);                   // the word now at the cursor
            break;
          }
        }
        found = true;
        cur[o] = c;
        nxw[o] = w;
      }
    }
    // x = logit + lambda L(h, y), in place
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      float4 l4 = lw[g];
      if (found) {
        const float4 d4 = *(const float4 *)(&D[256 * g + 4 * lane]);
        l4.x += d4.x;
        l4.y += d4.y;
        l4.z += d4.z;
        l4.w += d4.w;
      }
      val[4 * g] += l4.x;
      val[4 * g + 1] += l4.y;
      val[4 * g + 2] += l4.z;
      val[4 * g + 3] += l4.w;
    }
    if (found) {                              // the delta tile back to zero
#pragma unroll
      for (int g = 0; g < NG; ++g) *(float4 *)(&D[256 * g + 4 * lane]) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (allowed) {                            // constraint: disallowed words leave the candidates
      const uint32_t *aw = allowed + (size_t)s * ((V + 31) >> 5);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int c = vb + 256 * g + 4 * lane;
        const uint32_t w = c < Vr ? aw[c >> 5] : 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (!((w >> ((c + e) & 31)) & 1u)) val[4 * g + e] = -INFINITY;
      }
    }
    if (eosx && eos >= vb && eos < vb + SC_TV) {   // the row's EOS candidate, for the backoff stack
#pragma unroll
      for (int e = 0; e < 4 * NG; ++e)
        if (colv(e) == eos) eosx[row] = val[e];
    }

    // 3. candidates: x >= the running K-th value, and while the list is not
    //    full x >= a lower bound on this tile's K-th largest (G >= K lane
    //    groups: the smallest group maximum).  Each is inserted in turn into
    //    the running list (lanes 0 .. K-1, best first): its position is the
    //    number of entries better than it under (x desc, word asc), a total
    //    order; the entries from there on move down one lane and the last one
    //    leaves the list.
    float xm = val[0];
#pragma unroll
    for (int e = 1; e < 4 * NG; ++e) xm = fmaxf(xm, val[e]);
    const float thr = tr != -INFINITY ? tr : fmaxf(-__FLT_MAX__, group_bound(xm, G));
    if (__ballot(xm >= thr)) {
#pragma unroll
      for (int e = 0; e < 4 * NG; ++e) {
        uint64_t bal = __ballot(val[e] >= thr);
        while (bal) {
          const int j = (int)__builtin_ctzll(bal);
          bal &= bal - 1;
          const float cx = rdlane_f(val[e], j);
          const int cv = vb + 256 * (e >> 2) + 4 * j + (e & 3);   // the column of lane j's element e
          const int pos = __popcll(__ballot(lane < K && better(rx, rv, cx, cv)));
          if (pos < K) {
            const float ux = dpp_f<kDppShr1>(rx);
            const int uv = dpp_i<kDppShr1>(rv);
            if (lane > pos) {
              rx = ux;
              rv = uv;
            }
            if (lane == pos) {
              rx = cx;
              rv = cv;
            }
          }
        }
      }
      // the K-th value of the list (-inf while fewer than K)
      const float kx = rdlane_f(rx, K - 1);
      const int kv = rdlane_i(rv, K - 1);
      tr = kv >= 0 ? kx : -INFINITY;
    }

    if (jt == nt - 1) {
      // the row's last tile: partials reduced over the wave, and its list
      const size_t o = (size_t)row * nstrips + strip;
      const float m = wave_max(mr);
      float sg = mr == -INFINITY ? 0.f : sr * __expf(mr - m);
      sg = wave_sum(sg);
      if (lane == 0) stats[o] = make_float2(m, sg);
      if (lane < K) topk[o * K + lane] = Cand{rx, rv};
    }
  }
}

// ---------------------------------------------------------------------------
// Fused projection + score pass
// ---------------------------------------------------------------------------
// One workgroup = one block of 256 rows (sentence x beam) x one score strip
// (NT tiles of 256 columns).  Each tile's logits come out of the MFMA main loop
// and never reach HBM: the tile is staged through the (then idle) pipeline LDS
// a quarter of 64 rows at a time, and each row's eight threads (32 columns
// each) then
//   1. fold the tile into their running log-softmax partials (max, sum exp)
//      of the row (EOS bias included),
//   2. build lambda * L for their columns (Eq. 2): theta0 everywhere, the
//      unigram posteriors of the sentence's unigram range for the tile, and the
//      order 2..4 successors of the row's histories, in that order, so that
//      the sum is formed in a fixed order,
//   3. keep the values x = logit + lambda * L that can still enter the row's
//      top K: those >= a lower bound of the tile's K-th value (the smallest of
//      G >= K group maxima, every group maximum being a distinct element) and
//      above the running K-th value of the strip,
//   4. rank the kept values together with the running list (64-bit keys, one
//      compare per pair: x descending, then word ascending) and keep the K
//      best, spread over the row's eight threads (slots j and j + 8).
// The per-(row, strip) results have the layout of the score pass, so the
// merge is shared.  All of a row's LDS traffic stays inside its 8-lane group,
// i.e. inside one wave, whose LDS operations execute in program order.
constexpr int FS_COLS = 256;        // columns per tile
constexpr int kComputeUnits = 256;  // MI355X
constexpr int FS_SLOT_EL = 16;      // buffer: slots 0..15 the ranked output, then candidates and the running list

struct FsRowMeta {
  int base[3];                      // order 2..4 successor lists: first entry of the strip
  uint16_t b[3][LMBR_MAX_NT + 1];   // ... and each tile's range, relative to base
  const int2 *entries;              // the row's sentence: successor entries
  const float *ud;                  // ... dense history-free part of lambda * L
  float eos_b;                      // ... EOS bias
  int orig;                         // the row's index in the beam (s * K + k)
};

// Staged tile of 64 rows x 256 columns.  Row r takes 2 KB: its fp32 logits
// (later x) in the first KB and lambda * L (later the row's candidate buffer)
// in the second, so one base address plus immediate offsets reaches both.
// Float index of column c of row r in the first KB: 16-byte chunk k = c / 4
// sits at k ^ h(r, k).  A thread's eight chunks (its 32 columns) stay
// contiguous, reads take eight segments of two rows per 16-lane phase, and
// writes from the MFMA layout take 32 columns of rows r and r + 4: both are
// conflict-free with 64 banks.
__device__ __forceinline__ int fs_h(int r, int k) {
  return ((k >> 4) & 3) | ((r & 1) << 2) | (((r >> 2) & 1) << 3);
}
__device__ __forceinline__ int fs_idx(int r, int c) {
  const int k = c >> 2;
  return r * 512 + ((k ^ fs_h(r, k)) << 2) + (c & 3);
}
constexpr int FS_LOFF = 256;        // float offset of lambda * L within a row

// reductions over aligned groups of eight lanes
__device__ __forceinline__ float g8_min(float x) {
  x = fminf(x, dpp_f<kDppXor1>(x));
  x = fminf(x, dpp_f<kDppXor2>(x));
  return fminf(x, dpp_f<kDppHalfMirror>(x));
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
  // every pattern used stays inside a row of 16 lanes: no lane is out of range
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)x, CTRL, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(x >> 32), CTRL, 0xF, 0xF, true);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t g8_max_u64(uint64_t x) {
  uint64_t o = dpp_u64<kDppXor1>(x);
  x = o > x ? o : x;
  o = dpp_u64<kDppXor2>(x);
  x = o > x ? o : x;
  o = dpp_u64<kDppHalfMirror>(x);
  return o > x ? o : x;
}
// DPP16 row_shr:n (lane i takes lane i - n of its row of 16)
constexpr int kDppShr2 = 0x112, kDppShr4 = 0x114;
// exclusive prefix sum over an aligned group of eight lanes (g = lane % 8)
__device__ __forceinline__ int g8_excl_sum(int x, int g) {
  int s = x;
  int t = dpp_i<kDppShr1>(s);
  s += g >= 1 ? t : 0;
  t = dpp_i<kDppShr2>(s);
  s += g >= 2 ? t : 0;
  t = dpp_i<kDppShr4>(s);
  s += g >= 4 ? t : 0;
  return s - x;
}
__device__ __forceinline__ int g8_sum(int x) {
  x += dpp_i<kDppXor1>(x);
  x += dpp_i<kDppXor2>(x);
  return x + dpp_i<kDppHalfMirror>(x);
}
// Key of lane (this ^ R) within an aligned group of eight lanes (R = 1..7):
// quad_perm xor 1 / 2 / 3, row_half_mirror (xor 7), and their compositions.
constexpr int kDppXor3 = 0x1B;
template <int R>
__device__ __forceinline__ uint64_t g8_xor_u64(uint64_t x) {
  if constexpr (R == 1) return dpp_u64<kDppXor1>(x);
  else if constexpr (R == 2) return dpp_u64<kDppXor2>(x);
  else if constexpr (R == 3) return dpp_u64<kDppXor3>(x);
  else if constexpr (R == 7) return dpp_u64<kDppHalfMirror>(x);
  else if constexpr (R == 4) return dpp_u64<kDppHalfMirror>(dpp_u64<kDppXor3>(x));
  else if constexpr (R == 5) return dpp_u64<kDppHalfMirror>(dpp_u64<kDppXor2>(x));
  else return dpp_u64<kDppHalfMirror>(dpp_u64<kDppXor1>(x));
}
// Ranks (number of greater keys) of the S keys held by each lane of an 8-lane
// group among all 8 S keys of the group.
template <int S, int R>
__device__ __forceinline__ void g8_rank_step(const uint64_t (&k)[S], int (&rank)[S]) {
  uint64_t p[S];
#pragma unroll
  for (int u = 0; u < S; ++u) p[u] = g8_xor_u64<R>(k[u]);
#pragma unroll
  for (int u = 0; u < S; ++u)
#pragma unroll
    for (int v = 0; v < S; ++v) rank[u] += p[v] > k[u];
}
template <int S>
__device__ __forceinline__ void g8_rank(const uint64_t (&k)[S], int (&rank)[S]) {
#pragma unroll
  for (int u = 0; u < S; ++u) {
    rank[u] = 0;
#pragma unroll
    for (int v = 0; v < S; ++v)
      if (v != u) rank[u] += k[v] > k[u];
  }
  g8_rank_step<S, 1>(k, rank);
  g8_rank_step<S, 2>(k, rank);
  g8_rank_step<S, 3>(k, rank);
  g8_rank_step<S, 4>(k, rank);
  g8_rank_step<S, 5>(k, rank);
  g8_rank_step<S, 6>(k, rank);
  g8_rank_step<S, 7>(k, rank);
}
// (max, sum exp(. - max)) pairs
__device__ __forceinline__ void lse_merge(float &m, float &s, float mo, float so) {
  const float mx = fmaxf(m, mo);
  if (mx == -INFINITY) return;
  s = (m == -INFINITY ? 0.f : s * __expf(m - mx)) + (mo == -INFINITY ? 0.f : so * __expf(mo - mx));
  m = mx;
}
__device__ __forceinline__ void g8_lse(float &m, float &s) {
  lse_merge(m, s, dpp_f<kDppXor1>(m), dpp_f<kDppXor1>(s));
  lse_merge(m, s, dpp_f<kDppXor2>(m), dpp_f<kDppXor2>(s));
  lse_merge(m, s, dpp_f<kDppHalfMirror>(m), dpp_f<kDppHalfMirror>(s));
}

// Quarter q of the tile is accumulator block q of every wave: staged rows
// 0..31 are block rows 32q..32q+31, staged rows 32..63 are 128+32q.. .
// Register r of a lane is staged row R0 + 8 (r / 4) + r % 4 (R0 = 32 wm +
// 4 (lane / 32)): its chunk swizzle depends on r only through r % 2, so two
// base addresses per column block and immediate row offsets cover all 16.
template <int I, bool BIAS>
__device__ __forceinline__ void fs_stage(float *SA, const f32x16_t (&acc)[4][2], const float (&bcol)[2], int wm,
                                         int wn, int lane) {
  const int r0 = wm * 32 + 4 * (lane >> 5);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int c = wn * 64 + j * 32 + (lane & 31);
    float *b0 = SA + fs_idx(r0, c), *b1 = SA + fs_idx(r0 + 1, c) - 512;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float *b = (r & 1) ? b1 : b0;
      b[(8 * (r >> 2) + (r & 3)) * 512] = BIAS ? acc[I][j][r] + bcol[j] : acc[I][j][r];
    }
  }
}

__global__ __launch_bounds__(512)
void k_fused(const uint16_t *__restrict__ A, const uint16_t *__restrict__ Bw, const float *__restrict__ bias,
             int M, int V, int Kd, int K, int nMb, int nstrips, int NT, int remap,
             const int *__restrict__ ranges, const SentTable *__restrict__ tabs,
             const float *__restrict__ eos_bias, int eos, float lth0, float lth1, float lth2, float lth3,
             float lth4, const uint32_t *__restrict__ allowed, float *__restrict__ eosx,
             const double *__restrict__ q, float2 *__restrict__ stats, Cand *__restrict__ topk, int *err) {
  using S = TileShape<256, 256, 128, 64>;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[S::LDS_BYTES];
  __shared__ FsRowMeta rmeta[256];
  __shared__ int amap[256];
  __shared__ int wsum[8];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  int bid = blockIdx.x;
  if (remap) {
    const int per = (nMb * nstrips) >> 3;
    bid = (bid & 7) * per + (bid >> 3);
  }
  const int mb = bid % nMb, strip = bid / nMb;
  const int m0 = mb * 256;
  const int wm = wid / S::WAVES_N, wn = wid % S::WAVES_N;
  const int tile0 = strip * NT;
  const int nt = min(NT, ((V + FS_COLS - 1) / FS_COLS) - tile0);   // tiles of this strip

  // Live-row compaction: the block takes live rows m0 .. m0 + 255 in the
  // order of the live rows of the beam (a live row has a finite running
  // score); dead rows are neither projected nor scored.  Every workgroup
  // scans q itself (a block-wide prefix count over M rows).
  int nlive = 0;
  for (int c0 = 0; c0 < M; c0 += 512) {
    const int r = c0 + tid;
    const bool lv = r < M && q[r] != -INFINITY;
    const uint64_t bal = __ballot(lv);
    const int wpre = __builtin_amdgcn_mbcnt_hi((unsigned)(bal >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)bal, 0u));
    if (lane == 0) wsum[wid] = __popcll(bal);
    __syncthreads();
    int before = nlive, csum = 0;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      before += w < wid ? wsum[w] : 0;
      csum += wsum[w];
    }
    const int p = before + wpre;
    if (lv && p >= m0 && p < m0 + 256) amap[p - m0] = r;
    nlive += csum;
    __syncthreads();                                 // wsum is rewritten by the next chunk
  }
  const int nbl = min(256, nlive - m0);              // live rows of this block (uniform)
  if (nbl <= 0) return;
  if (tid < 256 && tid >= nbl) amap[tid] = amap[nbl - 1];   // a valid row for the GEMM's unused rows
  __syncthreads();

  // Per-row and per-sentence table ranges of this strip.  A successor list
  // longer than LMBR_DIR_MIN is preceded by its directory: ceil(V / 256) + 1
  // entry indices (first entry of each 256-column tile, then the end), packed
  // two per int2 in the Dt slots before the list; a shorter list is read here
  // and its words counted below each tile boundary.
  if (tid < 256) {
    FsRowMeta rm{};
    if (tid < nbl) {
      const int row = amap[tid];
      const int s = row / K;
      const SentTable tb = tabs[s];
      rm.orig = row;
      rm.entries = tb.entries;
      // dense layout: the row's own row of L (every order), no successor lists
      rm.ud = tb.dense ? tb.dense + (size_t)ranges[row * 6] * (size_t)(((V + 255) >> 8) << 8) : tb.uni_dense;
      rm.eos_b = eos_bias ? eos_bias[s] : 0.f;
      const int Dt = (((V + FS_COLS - 1) / FS_COLS) + 2) >> 1;
#pragma unroll
      for (int o = 0; o < 3; ++o) {
        if (tb.dense) continue;
        const int off = ranges[row * 6 + 2 * o], cnt = ranges[row * 6 + 2 * o + 1];
        if (cnt == 0) continue;
        if (!(off >= 0 && cnt > 0 && (int64_t)off + cnt <= (int64_t)tb.n_entries)) {
          flag_fault(err, LMBR_DEV_TABLE);
          continue;
        }
        rm.base[o] = off;
        if (cnt > LMBR_DIR_MIN && off >= Dt) {
          const uint32_t *dir = (const uint32_t *)(tb.entries + off - Dt);
          const uint32_t lo = min(max(dir[tile0], (uint32_t)off), (uint32_t)(off + cnt));
          rm.base[o] = (int)lo;
#pragma unroll
          for (int j = 0; j <= LMBR_MAX_NT; ++j) {
            const uint32_t d = j <= nt ? min(max(dir[tile0 + j], lo), (uint32_t)(off + cnt)) : lo;
            rm.b[o][j] = (uint16_t)min(d - lo, 65535u);
          }
        } else {
          int w[LMBR_DIR_MIN];
#pragma unroll
          for (int k = 0; k < LMBR_DIR_MIN; ++k) w[k] = k < cnt ? tb.entries[off + k].x : 0x7FFFFFFF;
#pragma unroll
          for (int j = 0; j <= LMBR_MAX_NT; ++j) {
            const int bound = (tile0 + min(j, nt)) * FS_COLS;
            int c = 0;
#pragma unroll
            for (int k = 0; k < LMBR_DIR_MIN; ++k) c += w[k] < bound;
            rm.b[o][j] = (uint16_t)c;
          }
        }
      }
    }
    rmeta[tid] = rm;
  }

  float *SA = (float *)smem;                         // [64 rows][2 KB]: logits then x | lambda * L then buffer

  // running state of this thread's row in each quarter
  float rs_m[4], rs_s[4];
  uint64_t rk0[4], rk1[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    rs_m[i] = -INFINITY;
    rs_s[i] = 0.f;
    rk0[i] = 0;
    rk1[i] = 0;
  }

  lds_sync_barrier();                                // the metadata is in LDS
  asm volatile("" ::"s"(bias), "s"(stats), "s"(topk), "s"(lth2), "s"(lth3), "s"(lth4));
  for (int jn = 0; jn < nt; ++jn) {
    const int n0 = (tile0 + jn) * FS_COLS;
    f32x16_t acc[4][2];
    mma_tile<256, 256, 128, 64>(A, Bw, M, V, Kd, m0, n0, (uint32_t)(uintptr_t)(lds_ptr_t)smem, wid, lane, acc,
                                amap);
    float bcol[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + (lane & 31);
      bcol[j] = (bias != nullptr && col < V) ? bias[col] : 0.f;
    }
    const bool partial = n0 + FS_COLS > V;

    auto quarter = [&](auto qd_c) {
      constexpr int qd = decltype(qd_c)::value;
      // per-lane layout values, rederived here (not kept live through the main loop)
      int t = tid, wq = wid;
      asm volatile("" : "+v"(t), "+s"(wq));
      const int er = t >> 3, ej = t & 7;             // row of the quarter, 32-column segment
      const int cb = n0 + ej * 32;                   // this thread's first column
      // this thread's eight chunks (its 32 columns): logical chunk q (columns
      // cb + 4q ..) sits at physical chunk (8 ej + q) ^ hh; lanes walking q in
      // step keep the 16-lane phases on distinct banks
      const int hh = fs_h(er, ej * 8);
      float *rowp = SA + er * 512;
      auto own = [&](int q) { return rowp + ((((ej * 8) + q) ^ hh) << 2); };
      const int swz = (er & 7) << 2;                 // buffer slot swizzle (rows of a wave on distinct banks)
      uint64_t *buf = (uint64_t *)(SA + er * 512 + FS_LOFF);
      const int rl = (er >> 5) * 128 + qd * 32 + (er & 31);
      const bool live = rl < nbl;
      const int row = live ? rmeta[rl].orig : 0;    // the row in the beam

      lds_sync_barrier();                            // main loop / previous quarter done with the buffers
      if (bias) fs_stage<qd, true>(SA, acc, bcol, wm, wn, lane);
      else fs_stage<qd, false>(SA, acc, bcol, wm, wn, lane);

      // the row's tables; the first successor of each order in the strip
      const int2 *ent = nullptr;
      const float *ud = nullptr;
      float eb = 0.f;
      int2 pf[3][2];
      int e0[3], e1[3];
#pragma unroll
      for (int o = 0; o < 3; ++o) {
        pf[o][0] = pf[o][1] = make_int2(-1, 0);
        e0[o] = e1[o] = 0;
      }
      if (live) {
        const FsRowMeta &rm = rmeta[rl];            // read in place (tile index is dynamic)
        ent = rm.entries;
        ud = rm.ud;
        eb = rm.eos_b;
#pragma unroll
        for (int o = 0; o < 3; ++o) {
          e0[o] = rm.base[o] + rm.b[o][jn];
          e1[o] = rm.base[o] + rm.b[o][jn + 1];
          if (e0[o] + ej < e1[o]) pf[o][0] = ent[e0[o] + ej];
          if (e0[o] + ej + 8 < e1[o]) pf[o][1] = ent[e0[o] + ej + 8];
        }
      }
      // history-free lambda * L of the wave's eight rows, straight from the
      // dense row into their L halves (one 1 KB row per load instruction:
      // lane l fills physical chunk l, i.e. logical chunk l ^ h)
      {
        const uint64_t udp = (uint64_t)(uintptr_t)ud;
        const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int eri = wq * 8 + i;
          const int rli = (eri >> 5) * 128 + qd * 32 + (eri & 31);
          if (rli < nbl) {
            const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)udp, 8 * i);
            const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(udp >> 32), 8 * i);
            const float *src = (const float *)(uintptr_t)(((uint64_t)hi << 32) | lo) + n0 +
                               4 * (lane ^ fs_h(eri, lane));
            asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src),
                         "{m0}"(lds0 + (uint32_t)(eri * 2048 + 1024))
                         : "memory");
          }
        }
      }
      lds_sync_barrier();                            // staged logits visible

      if (live) {
        if (eos >= cb && eos < cb + 32) SA[fs_idx(er, eos - n0)] += eb;
        float xv[32];                                // columns cb .. cb + 31
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float4 a = *(const float4 *)own(q);
          xv[4 * q] = a.x;
          xv[4 * q + 1] = a.y;
          xv[4 * q + 2] = a.z;
          xv[4 * q + 3] = a.w;
        }
        if (partial) {
#pragma unroll
          for (int k = 0; k < 32; ++k)
            if (cb + k >= V) xv[k] = -INFINITY;
        }
        // 1. log-softmax partials
        {
          float mt = xv[0];
#pragma unroll
          for (int k = 1; k < 32; ++k) mt = fmaxf(mt, xv[k]);
          const float mx = fmaxf(rs_m[qd], mt);
          if (mx != -INFINITY) {
            // exp(x - mx) = 2^(x log2 e - mx log2 e): one FMA and v_exp_f32 per value
            constexpr float kL2E = 1.44269504088896341f;
            const float nm = -mx * kL2E;
            float sacc = rs_m[qd] == -INFINITY ? 0.f : rs_s[qd] * __builtin_amdgcn_exp2f(fmaf(rs_m[qd], kL2E, nm));
#pragma unroll
            for (int k = 0; k < 32; ++k) sacc += __builtin_amdgcn_exp2f(fmaf(xv[k], kL2E, nm));
            rs_s[qd] = sacc;
            rs_m[qd] = mx;
          }
        }
        // 2. the order 2..4 terms of lambda * L on top of the history-free
        // row, order by order (LDS adds of one wave apply in issue order; a
        // successor's word is unique within its order), then x = logit +
        // lambda * L (also written back: later steps index it per column)
        wait_vmcnt<0>();
#pragma unroll
        for (int o = 0; o < 3; ++o) {
          const float lt = o == 0 ? lth2 : (o == 1 ? lth3 : lth4);
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const int c = pf[o][u].x - n0;
            if ((unsigned)c < (unsigned)FS_COLS) atomicAdd(&SA[fs_idx(er, c) + FS_LOFF], lt * __int_as_float(pf[o][u].y));
          }
          for (int e = e0[o] + ej + 16; e < e1[o]; e += 8) {
            const int2 en = ent[e];
            const int c = en.x - n0;
            if ((unsigned)c < (unsigned)FS_COLS) atomicAdd(&SA[fs_idx(er, c) + FS_LOFF], lt * __int_as_float(en.y));
          }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float4 l4 = *(const float4 *)(own(q) + FS_LOFF);
          xv[4 * q] += l4.x;
          xv[4 * q + 1] += l4.y;
          xv[4 * q + 2] += l4.z;
          xv[4 * q + 3] += l4.w;
        }
        if (allowed) {                               // constraint: disallowed words leave the candidates
          const uint32_t w = cb < V ? allowed[(size_t)(row / K) * ((V + 31) >> 5) + (cb >> 5)] : 0u;
#pragma unroll
          for (int k = 0; k < 32; ++k)
            if (!((w >> k) & 1u)) xv[k] = -INFINITY;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q)
          *(float4 *)own(q) = make_float4(xv[4 * q], xv[4 * q + 1], xv[4 * q + 2], xv[4 * q + 3]);
        if (eosx && eos >= cb && eos < cb + 32) eosx[row] = SA[fs_idx(er, eos - n0)];
        // 3. bounds and candidates
        float gmx[8];
#pragma unroll
        for (int g = 0; g < 8; ++g)
          gmx[g] = fmaxf(fmaxf(xv[4 * g], xv[4 * g + 1]), fmaxf(xv[4 * g + 2], xv[4 * g + 3]));
        float tau_t;
        {
          const float h0 = fmaxf(fmaxf(gmx[0], gmx[1]), fmaxf(gmx[2], gmx[3]));
          const float h1 = fmaxf(fmaxf(gmx[4], gmx[5]), fmaxf(gmx[6], gmx[7]));
          tau_t = g8_min(K <= 8 ? fmaxf(h0, h1) : fminf(h0, h1));
        }
        float tau_r = -INFINITY;
        if (jn > 0) {
          const uint64_t mine = (K - 1) >= 8 ? rk1[qd] : rk0[qd];
          const int hk = __shfl((int)(uint32_t)(mine >> 32), (lane & ~7) | ((K - 1) & 7));
          if (hk != 0) tau_r = unord_f((uint32_t)hk);
        }
        // kept: x >= tau_t and x > tau_r; positions by a prefix sum over the
        // row's eight lanes
        unsigned gm = 0;
#pragma unroll
        for (int g = 0; g < 8; ++g) gm |= (gmx[g] >= tau_t && gmx[g] > tau_r) ? (1u << g) : 0u;
        uint32_t km = 0;
#pragma unroll
        for (int g = 0; g < 8; ++g) {
          if (gm & (1u << g)) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              km |= xv[4 * g + i] >= tau_t && xv[4 * g + i] > tau_r ? (1u << (4 * g + i)) : 0u;
          }
        }
        const int mine_n = __popc(km);
        int pos = g8_excl_sum(mine_n, ej);
        int n = g8_sum(mine_n);
        // at most 32 keys per row are ranked (in registers, below): more
        // candidates than fit beside the running list take the exact path
        const int n_lim = 32 - (jn > 0 ? K : 0);
        if (n <= n_lim) {
          while (km) {
            const int k = __builtin_ctz(km);
            km &= km - 1;
            const float y = own(k >> 2)[k & 3];
            buf[(FS_SLOT_EL + pos) ^ swz] = cand_key(y, cb + k);
            ++pos;
          }
        }
        if (n > n_lim) {
          // many values at the bound (a strip's first tile, ties, few valid
          // columns): the tile's exact top K by K rounds of a row-wide argmax
          // over the values in registers
          uint32_t taken = 0;
          for (int r = 0; r < K; ++r) {
            uint64_t best = 0;
            int bi = -1;
#pragma unroll
            for (int k = 0; k < 32; ++k) {
              const float y = xv[k];
              const uint64_t kk = cand_key(y, cb + k);
              if (!((taken >> k) & 1u) && y != -INFINITY && kk > best) {
                best = kk;
                bi = k;
              }
            }
            const uint64_t w = g8_max_u64(best);
            if (bi >= 0 && best == w) taken |= 1u << bi;
            if (ej == 0) buf[(FS_SLOT_EL + r) ^ swz] = w;
          }
          n = K;
        }
        // 4. rank candidates and the running list together
        int N = n;
        if (jn > 0) {
          if (ej < K) buf[(FS_SLOT_EL + n + ej) ^ swz] = rk0[qd];
          if (ej + 8 < K) buf[(FS_SLOT_EL + n + ej + 8) ^ swz] = rk1[qd];
          N = n + K;
        }
        if (ej < K) buf[ej ^ swz] = 0;
        if (ej + 8 < K) buf[(ej + 8) ^ swz] = 0;
        // element f (f < N <= 32) belongs to lane f % 8 of the row: ranked in
        // registers across the row's lanes
        int nmax = N;                                // wave-wide (inactive lanes read as 0)
        nmax = max(nmax, dpp_i<kDppHalfMirror>(nmax));
        nmax = max(nmax, dpp_i<kDppMirror>(nmax));
        nmax = max(max(rdlane_i(nmax, 0), rdlane_i(nmax, 16)), max(rdlane_i(nmax, 32), rdlane_i(nmax, 48)));
        auto rank_in_regs = [&](auto s_c) {
          constexpr int S = decltype(s_c)::value;
          uint64_t kk[S];
          int rk[S];
#pragma unroll
          for (int u = 0; u < S; ++u) kk[u] = ej + 8 * u < N ? buf[(FS_SLOT_EL + ej + 8 * u) ^ swz] : 0ull;
          g8_rank<S>(kk, rk);
#pragma unroll
          for (int u = 0; u < S; ++u)
            if (ej + 8 * u < N && rk[u] < K) buf[rk[u] ^ swz] = kk[u];
        };
        if (nmax <= 8) rank_in_regs(std::integral_constant<int, 1>{});
        else if (nmax <= 16) rank_in_regs(std::integral_constant<int, 2>{});
        else if (nmax <= 24) rank_in_regs(std::integral_constant<int, 3>{});
        else rank_in_regs(std::integral_constant<int, 4>{});       // N <= 32 (n_lim above)
        rk0[qd] = ej < K ? buf[ej ^ swz] : 0;
        rk1[qd] = ej + 8 < K ? buf[(ej + 8) ^ swz] : 0;

        if (jn == nt - 1) {
          float m = rs_m[qd], s = rs_s[qd];
          g8_lse(m, s);
          const size_t o = (size_t)row * nstrips + strip;
          if (ej == 0) stats[o] = make_float2(m, s);
          if (ej < K) topk[o * K + ej] = key_cand(rk0[qd]);
          if (ej + 8 < K) topk[o * K + ej + 8] = key_cand(rk1[qd]);
        }
      }
    };
    quarter(std::integral_constant<int, 0>{});
    quarter(std::integral_constant<int, 1>{});
    quarter(std::integral_constant<int, 2>{});
    quarter(std::integral_constant<int, 3>{});
    lds_sync_barrier();                              // epilogue done: the stage buffers may be refilled
  }
}

// ---------------------------------------------------------------------------
// Merge/select (TopB per sentence), EOS handling, realignment, context probes
// ---------------------------------------------------------------------------
constexpr int MG_LIST = LMBR_MAX_TILES * LMBR_KMAX;   // per-wave staging of one row's lists
constexpr int MG_WAVES = 8;                            // waves per sentence: one row each for K <= 8

__global__ __launch_bounds__(MG_WAVES * 64)
void k_merge(int V, int K, int ntiles, int eos, int t_idx, int M,
             const float2 *__restrict__ stats, const Cand *__restrict__ topk,
             double *__restrict__ q, uint64_t *__restrict__ ctx, uint64_t *__restrict__ hh,
             int *__restrict__ len, int *__restrict__ ranges, int *__restrict__ bp,
             int *__restrict__ tok, double *__restrict__ qhist,
             const SentTable *__restrict__ tabs, StepOpts opt, int *__restrict__ parent_out,
             int *__restrict__ token_out, double *__restrict__ score_out) {
  __shared__ double s_q[LMBR_KMAX], s_lse[LMBR_KMAX];
  __shared__ float s_rx[LMBR_KMAX][LMBR_KMAX];
  __shared__ int s_rv[LMBR_KMAX][LMBR_KMAX];
  __shared__ uint64_t s_ctx[LMBR_KMAX], s_hh[LMBR_KMAX];
  __shared__ int s_len[LMBR_KMAX];
  __shared__ int s_selk[LMBR_KMAX], s_selv[LMBR_KMAX];
  __shared__ double s_sels[LMBR_KMAX];
  __shared__ uint64_t s_nctx[LMBR_KMAX];
  __shared__ int s_nlen[LMBR_KMAX], s_live[LMBR_KMAX];
  __shared__ Cand s_list[MG_WAVES][MG_LIST];

  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  // a row's tile partials and (when they fit four per lane) its per-tile
  // lists, loaded one row ahead of their use; the wave's first row is loaded
  // together with the beam state below
  const int nl = ntiles * K;
  const bool fit = nl <= 256;
  auto load_row = [&](int k, float2 &a, float2 &b, Cand (&c)[4]) {
    const int row = s * K + k;
    a = lane < ntiles ? stats[(size_t)row * ntiles + lane] : make_float2(-INFINITY, 0.f);
    b = lane + 64 < ntiles ? stats[(size_t)row * ntiles + lane + 64] : make_float2(-INFINITY, 0.f);
    if (fit) {
      const Cand *src = topk + (size_t)row * nl;
#pragma unroll
      for (int u = 0; u < 4; ++u) c[u] = 64 * u + lane < nl ? src[64 * u + lane] : Cand{-INFINITY, -1};
    }
  };
  float2 pa = make_float2(-INFINITY, 0.f), pb = pa;
  Cand pc[4];
  if (wid < K) load_row(wid, pa, pb, pc);
  if (tid < K) {
    const int row = s * K + tid;
    s_q[tid] = q[row];
    s_ctx[tid] = ctx[row];
    s_hh[tid] = hh[row];
    s_len[tid] = len[row];
    s_selk[tid] = 0;
    s_selv[tid] = 0;
    s_sels[tid] = -INFINITY;
  }
  __syncthreads();

  // each row: log-sum-exp over its tiles, and its K best by merging the
  // per-tile sorted lists (staged in LDS; list heads held by lanes)
  Cand *L = s_list[wid];
  for (int k = wid; k < K; k += MG_WAVES) {
    const int row = s * K + k;
    const float2 a = pa, b = pb;
    Cand cl[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) cl[u] = pc[u];
    if (k + MG_WAVES < K) load_row(k + MG_WAVES, pa, pb, pc);
    if (s_q[k] == -INFINITY) {
      if (lane < K) {
        s_rx[k][lane] = -INFINITY;
        s_rv[k][lane] = -1;
      }
      if (lane == 0) s_lse[k] = 0.0;
      continue;
    }
    const float m = wave_max(fmaxf(a.x, b.x));
    float sg = (a.x != -INFINITY ? a.y * __expf(a.x - m) : 0.f) + (b.x != -INFINITY ? b.y * __expf(b.x - m) : 0.f);
    sg = wave_sum(sg);
    if (lane == 0) {
      const double lse = (double)m + log((double)sg);
      s_lse[k] = lse;
      // a NaN or +inf logit makes the normaliser non-finite
      if (!isfinite(lse)) flag_fault(opt.err, LMBR_DEV_NONFINITE);
    }

    if (fit) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (64 * u + lane < nl) L[64 * u + lane] = cl[u];
    } else {
      const Cand *src = topk + (size_t)row * nl;
      for (int i = lane; i < nl; i += 64) L[i] = src[i];
    }
    int p0 = 0, p1 = 0;
    for (int r = 0; r < K; ++r) {
      float hx = -INFINITY;
      int hv = 0x7FFFFFFF, which = -1;
      if (lane < ntiles && p0 < K) {
        const Cand c = L[lane * K + p0];
        if (c.v >= 0) { hx = c.x; hv = c.v; which = 0; }
      }
      if (lane + 64 < ntiles && p1 < K) {
        const Cand c = L[(lane + 64) * K + p1];
        if (c.v >= 0 && better(c.x, c.v, hx, hv)) { hx = c.x; hv = c.v; which = 1; }
      }
      float wx = hx;
      int wv = hv;
      wave_argmax(wx, wv);
      if (which >= 0 && hv == wv) {
        if (which == 0) ++p0;
        else ++p1;
      }
      if (lane == 0) {
        s_rx[k][r] = wx;
        s_rv[k][r] = (wv == 0x7FFFFFFF) ? -1 : wv;
      }
    }
  }
  __syncthreads();

  // TopB over the sentence: score = q_k + (x - lse_k) in fp64, ties by k*V + v
  if (wid == 0) {
    int p = 0, nsel = 0;
    for (int r = 0; r < K; ++r) {
      double sc = -INFINITY;
      int flat = 0x7FFFFFFF;
      if (lane < K && p < K && s_rv[lane][p] >= 0 && s_q[lane] != -INFINITY) {
        sc = s_q[lane] + ((double)s_rx[lane][p] - s_lse[lane]);
        flat = lane * V + s_rv[lane][p];
      }
      double wsc = sc;
      int wfl = flat;
      wave_argmax_d(wsc, wfl);
      if (wsc == -INFINITY || wfl == 0x7FFFFFFF) break;
      if (lane < K && flat == wfl) ++p;
      if (lane == 0) {
        s_selk[r] = wfl / V;
        s_selv[r] = wfl % V;
        s_sels[r] = wsc;
      }
      ++nsel;
    }
    // fewer finite candidates than slots: the remaining slots take the -inf
    // candidates in flat-index order (every column of a dead row; the
    // disallowed columns of a live row under a constraint)
    if (lane == 0) {
      const uint32_t *aw = opt.allowed ? opt.allowed + (size_t)s * ((V + 31) >> 5) : nullptr;
      int r = nsel;
      for (int k = 0; k < K && r < K; ++k) {
        const bool dead = s_q[k] == -INFINITY;
        if (!dead && !aw) continue;
        // a live row here has fewer than K allowed words: the scan is short
        for (int v = 0; v < V && r < K; ++v) {
          if (!dead && ((aw[v >> 5] >> (v & 31)) & 1u)) continue;
          s_selk[r] = k;
          s_selv[r] = v;
          s_sels[r] = -INFINITY;
          ++r;
        }
      }
    }
  }
  __syncthreads();

  // EOS candidates of live rows that TopB did not keep: the sentence keeps the
  // best of them over all steps (score, or score per word; then earlier step,
  // then lower parent slot), returned when no hypothesis finishes
  const int t1 = t_idx + 1;
  if (opt.backup && tid == 0) {
    double bs = opt.sent[s].backup_score;
    int bt = opt.sent[s].backup_step, bk = opt.sent[s].backup_slot;
    for (int k = 0; k < K; ++k) {
      if (s_q[k] == -INFINITY) continue;
      const float ex = opt.eosx[s * K + k];
      if (ex == -INFINITY) continue;
      bool kept = false;
      for (int j = 0; j < K; ++j) kept |= s_selk[j] == k && s_selv[j] == eos;
      if (kept) continue;
      const double c = s_q[k] + ((double)ex - s_lse[k]);
      if (c == -INFINITY) continue;
      const bool take = bt == 0 || (opt.length_norm ? c / t1 > bs / bt : c > bs);
      if (take) {
        bs = c;
        bt = t1;
        bk = k;
      }
    }
    opt.sent[s].backup_score = bs;
    opt.sent[s].backup_step = bt;
    opt.sent[s].backup_slot = bk;
  }

  if (tid < K) {
    const int j = tid, k = s_selk[j], v = s_selv[j];
    const double sc = s_sels[j];
    const int row = s * K + j;
    const size_t hidx = (size_t)t_idx * M + row;
    if (isnan(sc)) flag_fault(opt.err, LMBR_DEV_NONFINITE);
    // early pruning: the best finished value including this step's EOS
    // entries; a live slot below it minus the width is dropped
    bool pruned = false;
    if (opt.prune) {
      auto value = [&](double x) { return opt.length_norm ? x / t1 : x; };
      double fb = opt.sent[s].best_final;
      for (int i = 0; i < K; ++i)
        if (s_selv[i] == eos && s_sels[i] != -INFINITY) fb = fmax(fb, value(s_sels[i]));
      pruned = sc != -INFINITY && v != eos && value(sc) < fb - opt.prune_width;
      if (j == 0) opt.sent[s].best_final = fb;
    }
    bp[hidx] = k;
    tok[hidx] = v;
    qhist[hidx] = pruned ? -INFINITY : sc;
    if (parent_out) parent_out[row] = k;
    if (token_out) token_out[row] = v;
    if (score_out) score_out[row] = sc;
    // EOS: pushed to F (qhist), then masked; the sentence's last step ends
    // every slot (the finished set reads them from qhist)
    const bool live = sc != -INFINITY && v != eos && !pruned && !(opt.steps && t1 >= opt.steps[s]);
    q[row] = live ? sc : -INFINITY;
    const uint64_t c = ((s_ctx[k] << 21) | (uint64_t)(v + 1)) & kCtxMaskDev;
    ctx[row] = c;
    hh[row] = mix64(s_hh[k] ^ (uint64_t)(v + 1));
    len[row] = s_len[k] + 1;
    s_nctx[j] = c;
    s_nlen[j] = s_len[k] + 1;
    s_live[j] = live;
  }
  __syncthreads();
  const SentTable &tb = tabs[s];
  if (tb.dense) {
    // dense layout: the row of L of each live slot (its longest history in
    // the table), in the first field; the others stay 0
    if (tid < K) {
      const int j = tid, row = s * K + j;
      ranges[row * 6] = s_live[j] ? dense_row(tb, s_nctx[j], s_nlen[j], opt.err) : 0;
#pragma unroll
      for (int f = 1; f < 6; ++f) ranges[row * 6 + f] = 0;
    }
  } else if (tid < 3 * K) {
    const int j = tid / 3, o = tid % 3;
    int2 r = make_int2(0, 0);
    if (s_live[j] && s_nlen[j] >= o + 1) r = probe(tb, s_nctx[j] & ((1ull << (21 * (o + 1))) - 1), opt.err);
    const int row = s * K + j;
    ranges[row * 6 + o * 2] = r.x;
    ranges[row * 6 + o * 2 + 1] = r.y;
  }
}

// ---------------------------------------------------------------------------
// GetBestHypothesis: best F entry per sentence, traced back through bp/tok
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64)
void k_traceback(int K, int M, int T_max, int tcur, int eos, StepOpts opt, const int *__restrict__ bp,
                 const int *__restrict__ tok, const double *__restrict__ qhist, int *__restrict__ tokens_out,
                 int *__restrict__ len_out, double *__restrict__ score_out,
                 int *__restrict__ step_out, int *__restrict__ slot_out) {
  const int s = blockIdx.x, lane = threadIdx.x;
  const int tend = opt.steps ? min(tcur, opt.steps[s]) : tcur;   // the sentence's last step
  // rank value: the score, or the score per word (an entry of 0-based step t holds t + 1 words)
  auto rankv = [&](double sc, int t) { return opt.length_norm ? sc / (t + 1) : sc; };
  double bs = -INFINITY;
  int bkey = 0x7FFFFFFF;                    // t * K + j: earlier step, then lower slot
  for (int i = lane; i < tend * K; i += 64) {
    const int t = i / K, j = i % K;
    const size_t idx = (size_t)t * M + s * K + j;
    const double sc = qhist[idx];
    if (tok[idx] == eos && sc != -INFINITY && better_d(rankv(sc, t), i, bs, bkey)) { bs = rankv(sc, t); bkey = i; }
  }
  if (!opt.backup && tend > 0) {            // slots live after the last step finish there
    for (int j = lane; j < K; j += 64) {
      const int key = (tend - 1) * K + j;
      const size_t idx = (size_t)(tend - 1) * M + s * K + j;
      const double sc = qhist[idx];
      if (tok[idx] != eos && sc != -INFINITY && better_d(rankv(sc, tend - 1), key, bs, bkey)) {
        bs = rankv(sc, tend - 1);
        bkey = key;
      }
    }
  }
  wave_argmax_d(bs, bkey);
  const int found = bs != -INFINITY;
  int bt = found ? bkey / K : -1, j = found ? bkey % K : -1;
  double score = found ? qhist[(size_t)bt * M + s * K + j] : -INFINITY;
  int last = bt;                            // last traced step
  int ended_eos = 0;
  if (!found && opt.backup) {
    const lmbr_sentence_record b = opt.sent[s];
    if (b.backup_step > 0) {                // the best EOS candidate that did not survive
      bt = b.backup_step - 1;
      j = b.backup_slot;
      score = b.backup_score;
      last = bt - 1;
      ended_eos = 1;
    }
  }
  for (int tt = lane; tt < T_max; tt += 64)
    if (tt > bt) tokens_out[(size_t)s * T_max + tt] = -1;
  if (lane == 0) {
    if (slot_out) slot_out[s] = j;
    if (step_out) step_out[s] = bt;
    len_out[s] = bt + 1;
    score_out[s] = score;
    if (ended_eos) tokens_out[(size_t)s * T_max + bt] = eos;
    for (int tt = last; tt >= 0; --tt) {
      j = min(max(j, 0), K - 1);
      const size_t idx = (size_t)tt * M + s * K + j;
      tokens_out[(size_t)s * T_max + tt] = tok[idx];
      j = bp[idx];
    }
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_synth_hidden(const uint64_t *hh, uint16_t *hidden, int M, int H, hipStream_t st) {
  const int threads = 128;
  const int bpr = (H / 8 + threads - 1) / threads;     // workgroups per row
  hipLaunchKernelGGL(k_synth_hidden, dim3((unsigned)((int64_t)M * bpr)), dim3(threads), 0, st, hh, hidden, M,
                     H, bpr);
  return hipGetLastError();
}

hipError_t launch_state_init(int B, int K, uint64_t seed, double *q, uint64_t *ctx, uint64_t *hh,
                             int *len, int *ranges, lmbr_sentence_record *sent, hipStream_t st) {
  const int n = B * K;
  hipLaunchKernelGGL(k_state_init, dim3((n + 255) / 256), dim3(256), 0, st, B, K, seed, q, ctx, hh, len,
                     ranges, sent);
  return hipGetLastError();
}

hipError_t launch_state_probe(int B, int K, const SentTable *tabs, const double *q, const uint64_t *ctx,
                              const int *len, int *ranges, int *err, hipStream_t st) {
  const int n = B * K * 3;
  hipLaunchKernelGGL(k_state_probe, dim3((n + 255) / 256), dim3(256), 0, st, B, K, tabs, q, ctx, len,
                     ranges, err);
  return hipGetLastError();
}

hipError_t launch_transpose_bf16(const uint16_t *src, uint16_t *dst, int rows, int cols, hipStream_t st) {
  hipLaunchKernelGGL(k_transpose_bf16, dim3((cols + 31) / 32, (rows + 31) / 32), dim3(256), 0, st, src,
                     dst, rows, cols);
  return hipGetLastError();
}

hipError_t launch_gather_rows(void *dst, const void *src, const int *rows, int n, int64_t row_bytes,
                              hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather_rows, dim3(n), dim3(256), 0, st, (uint32_t *)dst, (const uint32_t *)src, rows,
                     n, row_bytes / 4);
  return hipGetLastError();
}

GemmPlan gemm_plan(int M, int N) {
  GemmPlan p{};
  if (M > 512) {
    p.bm = 256; p.bn = 256; p.threads = 512;
  } else if (M > 64) {
    p.bm = 128; p.bn = 128; p.threads = 256;
  } else {
    p.bm = 64; p.bn = 128; p.threads = 256;
  }
  p.nMb = (M + p.bm - 1) / p.bm;
  p.nNb = (N + p.bn - 1) / p.bn;
  // strips of NT column tiles per workgroup: the fewest tiles per workgroup
  // that still fit the grid in one round over the CUs.  With one or two row
  // blocks a workgroup keeps one tile: when sentences finish, the blocks of
  // dead rows exit and the other block's tiles spread over every CU (base
  // workload, half the batch finished: 48.0 -> 45.1 us per decode step)
  p.nt = 1;
  while (p.nMb >= 3 && p.nMb * ((p.nNb + p.nt - 1) / p.nt) > kComputeUnits) ++p.nt;
  const int nstrips = (p.nNb + p.nt - 1) / p.nt;
  p.remap = ((p.nMb * nstrips) % 8 == 0) ? 1 : 0;
  return p;
}

hipError_t launch_gemm(const uint16_t *A, const uint16_t *Bw, const float *bias, float *C, int M, int N,
                       int Kd, int64_t ldc, const double *q, int *live_count, hipStream_t st) {
  const GemmPlan p = gemm_plan(M, N);
  const dim3 grid((unsigned)(p.nMb * ((p.nNb + p.nt - 1) / p.nt)));
  if (p.bm == 256) {
    // eight waves of 128 x 64; the 128 KB of stages allow one workgroup per CU
    hipLaunchKernelGGL((k_gemm<256, 256, 128, 64>), grid, dim3(512), 0, st, A, Bw, bias, C, M, N, Kd, ldc,
                       p.nMb, p.nNb, p.nt, p.remap, q, live_count);
  } else if (p.bm == 128) {
    hipLaunchKernelGGL((k_gemm<128, 128, 64, 64>), grid, dim3(256), 0, st, A, Bw, bias, C, M, N, Kd, ldc,
                       p.nMb, p.nNb, p.nt, p.remap, q, live_count);
  } else {
    hipLaunchKernelGGL((k_gemm<64, 128, 32, 64>), grid, dim3(256), 0, st, A, Bw, bias, C, M, N, Kd, ldc,
                       p.nMb, p.nNb, p.nt, p.remap, q, live_count);
  }
  return hipGetLastError();
}

hipError_t launch_add_scalar(float *x, size_t n, float c, hipStream_t st) {
  const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_add_scalar, dim3(std::max(blocks, 1u)), dim3(256), 0, st, x, n, c);
  return hipGetLastError();
}


ScorePlan score_plan(int B, int K, int V) {
  ScorePlan p{};
  const int M = B * K;
  auto tiles = [&](int tv) { return (V + tv - 1) / tv; };
  // The score pass: a workgroup per (sentence, strip of 1024-column tiles),
  // five per CU at a time.  The strips are cut for about two rounds of
  // workgroups over the CUs: shorter strips spread the work wider and even
  // out the tail, longer ones tighten each row's running K-th value and share
  // the per-strip set-up.  A strip keeps at least two tiles while that still
  // leaves two workgroups per CU (one-tile strips measured 33% slower at
  // 768 rows and 7% at 256).  At the large workload this gives 9 strips of 7
  // tiles, 8% faster than 4 of 16.  The merge sees at most LMBR_MAX_TILES.
  p.ntiles = tiles(SC_TV);
  const int want = (10 * kComputeUnits + B - 1) / B;   // strips per sentence
  int snt = std::max(1, (p.ntiles + want - 1) / want);
  if (snt < 2 && p.ntiles >= 2 && (p.ntiles + 1) / 2 * B >= 2 * kComputeUnits) snt = 2;
  while ((p.ntiles + snt - 1) / snt > LMBR_MAX_TILES) ++snt;
  p.score_nt = snt;
  p.score_strips = (p.ntiles + snt - 1) / snt;
  // The fused pass keeps a row's running top-K over a strip of tiles: longer
  // strips tighten the running bound (fewer candidates to rank) and share the
  // per-strip set-up and output, shorter strips make more workgroups.  Halve
  // the strip (from LMBR_MAX_NT tiles) while the workgroups still fit in one
  // round over the CUs (a partial second round measured slower than longer
  // strips), with at most LMBR_MAX_TILES strips.
  const int t256 = tiles(FS_COLS), nMb = (M + 255) / 256;
  int nt = LMBR_MAX_NT;
  while (nt > 1) {
    const int half = (t256 + nt / 2 - 1) / (nt / 2);
    if (half > LMBR_MAX_TILES || nMb * half > kComputeUnits) break;
    nt /= 2;
  }
  p.fused_nt = nt;
  p.fused_strips = (t256 + nt - 1) / nt;
  return p;
}

hipError_t launch_score(const ScorePlan &p, const float *logits, int64_t ld, int B, int V, int K,
                        const double *q, const int *ranges, const SentTable *tabs, const float *eos_bias,
                        int eos, float lam, const float *theta, const uint32_t *allowed, float *eosx,
                        float2 *stats, Cand *topk, int *err, hipStream_t st) {
  const dim3 grid((unsigned)p.score_strips, (unsigned)B);
  int G = 1;
  while (G < K) G <<= 1;
#define LMBR_SCORE_ARGS                                                                                   \
  logits, ld, V, K, p.ntiles, p.score_nt, p.score_strips, G, q, ranges, tabs, eos_bias, eos, lam * theta[2], \
      lam * theta[3], lam * theta[4], allowed, eosx, stats, topk, err
  hipLaunchKernelGGL(k_score, grid, dim3(SC_WAVES * 64), 0, st, LMBR_SCORE_ARGS);
#undef LMBR_SCORE_ARGS
  return hipGetLastError();
}

hipError_t launch_fused(const ScorePlan &p, const uint16_t *A, const uint16_t *Bw, const float *bias, int M,
                        int V, int Kd, int K, const int *ranges, const SentTable *tabs, const float *eos_bias,
                        int eos, float lam, const float *theta, const uint32_t *allowed, float *eosx,
                        const double *q, float2 *stats, Cand *topk, int *err, hipStream_t st) {
  const int NT = p.fused_nt;
  const int nMb = (M + 255) / 256;
  const int nblk = nMb * p.fused_strips;
  const int remap = (nblk % 8 == 0) ? 1 : 0;
  hipLaunchKernelGGL(k_fused, dim3((unsigned)nblk), dim3(512), 0, st, A, Bw, bias, M, V, Kd, K, nMb,
                     p.fused_strips, NT, remap, ranges, tabs, eos_bias, eos, lam * theta[0], lam * theta[1], lam * theta[2],
                     lam * theta[3], lam * theta[4], allowed, eosx, q, stats, topk, err);
  return hipGetLastError();
}

hipError_t launch_merge(int B, int V, int K, int ntiles, int eos, int t_idx, const float2 *stats,
                        const Cand *topk, double *q, uint64_t *ctx, uint64_t *hh, int *len, int *ranges,
                        int *bp, int *tok, double *qhist, const SentTable *tabs, const StepOpts &opt,
                        int *parent_out, int *token_out, double *score_out, hipStream_t st) {
  hipLaunchKernelGGL(k_merge, dim3(B), dim3(MG_WAVES * 64), 0, st, V, K, ntiles, eos, t_idx, B * K, stats, topk, q,
                     ctx, hh, len, ranges, bp, tok, qhist, tabs, opt, parent_out, token_out, score_out);
  return hipGetLastError();
}

hipError_t launch_traceback(int B, int K, int T_max, int tcur, int eos, const StepOpts &opt, const int *bp,
                            const int *tok, const double *qhist, int *tokens_out, int *len_out,
                            double *score_out, int *step_out, int *slot_out, hipStream_t st) {
  hipLaunchKernelGGL(k_traceback, dim3(B), dim3(64), 0, st, K, B * K, T_max, tcur, eos, opt, bp, tok, qhist,
                     tokens_out, len_out, score_out, step_out, slot_out);
  return hipGetLastError();
}

}  // namespace lmbr
