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

#include <cstdint>

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

__device__ __forceinline__ int lower_bound_tok(const int2 *e, int n, int v) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (e[mid].x < v) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Linear-probing lookup of a packed history; returns (offset, count) or (0, 0).
__device__ __forceinline__ int2 probe(const SentTable &tb, uint64_t key) {
  uint32_t h = (uint32_t)(mix64(key) & tb.mask);
  for (uint32_t step = 0; step <= tb.mask; ++step) {
    const Slot sl = tb.slots[h];
    if (sl.key == key) return make_int2((int)sl.off, (int)sl.cnt);
    if (sl.key == kEmptyKeyDev) break;
    h = (h + 1) & tb.mask;
  }
  return make_int2(0, 0);
}

// (x desc, v asc) "a ranks before b"
__device__ __forceinline__ bool better(float ax, int av, float bx, int bv) {
  return ax > bx || (ax == bx && av < bv);
}
__device__ __forceinline__ bool better_d(double ax, long long av, double bx, long long bv) {
  return ax > bx || (ax == bx && av < bv);
}

__device__ __forceinline__ void wave_argmax(float &x, int &v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ox = __shfl_xor(x, off, 64);
    const int ov = __shfl_xor(v, off, 64);
    if (better(ox, ov, x, v)) { x = ox; v = ov; }
  }
}

__device__ __forceinline__ void wave_argmax_d(double &x, long long &v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const double ox = __shfl_xor(x, off, 64);
    const long long ov = __shfl_xor(v, off, 64);
    if (better_d(ox, ov, x, v)) { x = ox; v = ov; }
  }
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

// Merge two (max, sum exp(x - max)) partials.
__device__ __forceinline__ void lse_combine(float &m, float &s, float om, float os) {
  if (om > m) { const float tm = m, ts = s; m = om; s = os; om = tm; os = ts; }
  if (om != -INFINITY) s += os * __expf(om - m);
}

}  // namespace dev

using namespace dev;

// ---------------------------------------------------------------------------
// Stand-in decoder state and beam-state bookkeeping
// ---------------------------------------------------------------------------
__global__ void k_synth_hidden(const uint64_t *__restrict__ hh, uint16_t *__restrict__ hidden,
                               int M, int H) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * H) return;
  const int m = (int)(i / H), c = (int)(i % H);
  hidden[i] = bf16_rne(irwin_hall(mix64(hh[m] + (uint64_t)c)));
}

__global__ void k_state_init(int B, int K, uint64_t seed, double *q, uint64_t *ctx, uint64_t *hh,
                             int *len, int *ranges) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * K) return;
  const int s = i / K, k = i % K;
  q[i] = k == 0 ? 0.0 : -INFINITY;
  ctx[i] = 0;
  hh[i] = mix64(mix64(seed + 0x48ull) ^ (uint64_t)s);
  len[i] = 0;
#pragma unroll
  for (int r = 0; r < 6; ++r) ranges[i * 6 + r] = 0;
}

__global__ void k_state_probe(int B, int K, const SentTable *__restrict__ tabs,
                              const double *__restrict__ q, const uint64_t *__restrict__ ctx,
                              const int *__restrict__ len, int *__restrict__ ranges) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * K * 3) return;
  const int row = i / 3, o = i % 3;          // order n = o + 2 needs n - 1 = o + 1 words
  int2 r = make_int2(0, 0);
  if (q[row] != -INFINITY && len[row] >= o + 1) {
    const uint64_t key = ctx[row] & ((1ull << (21 * (o + 1))) - 1);
    r = probe(tabs[row / K], key);
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

// ---------------------------------------------------------------------------
// Projection: bf16 MFMA GEMM, C[M, N] = A[M, Kd] . Bw[N, Kd]^T + bias
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
void k_gemm(const uint16_t *__restrict__ A, const uint16_t *__restrict__ Bw,
            const float *__restrict__ bias, float *__restrict__ C, int M, int N, int Kd,
            int64_t ldc, int nMb, int nNb, int remap) {
  constexpr int WAVES_N = BN / WN;
  constexpr int NT = (BM / WM) * WAVES_N * 64;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int BK = 64;                       // bf16 per row per stage: 8 chunks of 16 B
  constexpr int AC = BM * 8 / NT, BC = BN * 8 / NT;
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0, "tile/thread mismatch");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * BK];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int bid = blockIdx.x;
  if (remap) {
    // Consecutive workgroups land on different XCDs; give each XCD a contiguous
    // run of tiles so the M-blocks sharing a W block share that XCD's L2.
    const int per = (nMb * nNb) >> 3;
    bid = (bid & 7) * per + (bid >> 3);
  }
  const int mb = bid % nMb, nb = bid / nMb;
  const int m0 = mb * BM, n0 = nb * BN;
  const int wm = wid / WAVES_N, wn = wid % WAVES_N;

  u32x4_t ra[AC], rb[BC];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      const int qd = tid + i * NT, r = qd >> 3, c = qd & 7;
      const int gr = min(m0 + r, M - 1);
      ra[i] = *(const u32x4_t *)(A + (size_t)gr * Kd + kt * BK + c * 8);
    }
#pragma unroll
    for (int i = 0; i < BC; ++i) {
      const int qd = tid + i * NT, r = qd >> 3, c = qd & 7;
      const int gr = min(n0 + r, N - 1);
      rb[i] = *(const u32x4_t *)(Bw + (size_t)gr * Kd + kt * BK + c * 8);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      const int qd = tid + i * NT, r = qd >> 3, c = qd & 7;
      *(u32x4_t *)(&As[buf][r * BK + ((c ^ (r & 7)) << 3)]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BC; ++i) {
      const int qd = tid + i * NT, r = qd >> 3, c = qd & 7;
      *(u32x4_t *)(&Bs[buf][r * BK + ((c ^ (r & 7)) << 3)]) = rb[i];
    }
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = Kd / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int chunk = kk * 2 + (lane >> 5);
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WM + i * 32 + (lane & 31);
        af[i] = *(const bf16x8_t *)(&As[cur][r * BK + ((chunk ^ (r & 7)) << 3)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WN + j * 32 + (lane & 31);
        bfr[j] = *(const bf16x8_t *)(&Bs[cur][r * BK + ((chunk ^ (r & 7)) << 3)]);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // 32x32 accumulator layout: lane l holds column l % 32 and rows
  // 8 * (r / 4) + 4 * (l / 32) + r % 4 for r = 0..15.
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * WN + j * 32 + (lane & 31);
      const float bcol = (bias != nullptr && col < N) ? bias[col] : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < M && col < N) C[(size_t)row * ldc + col] = acc[i][j][r] + bcol;
      }
    }
}

// ---------------------------------------------------------------------------
// Fused score pass: log-softmax partials + LMBR add + per-row partial top-K
// ---------------------------------------------------------------------------
constexpr int SC_THREADS = 256;
constexpr int SC_CAP = 512;

template <int VPT>
__global__ __launch_bounds__(SC_THREADS)
void k_score(const float *__restrict__ logits, int64_t ld, int V, int K, int ntiles,
             const double *__restrict__ q, const int *__restrict__ ranges,
             const SentTable *__restrict__ tabs, const float *__restrict__ eos_bias, int eos,
             float lam, float th0, float th1, float th2, float th3, float th4,
             float2 *__restrict__ stats, Cand *__restrict__ topk) {
  constexpr int TV = SC_THREADS * VPT;
  constexpr int G = VPT / 4;                        // float4 groups per thread
  __shared__ __attribute__((aligned(16))) float Lsh[TV];   // theta0 + theta1 * p(unigram)
  __shared__ __attribute__((aligned(16))) float Dsh[TV];   // sum_{n>=2} theta_n * p, per row
  __shared__ float cx[SC_CAP];
  __shared__ int cv[SC_CAP];
  __shared__ int s_lohi[8];
  __shared__ int s_cnt;
  __shared__ float s_rf[8];
  __shared__ float s_rs[8];
  __shared__ int s_ri[8];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int tile = blockIdx.x, s = blockIdx.y;
  const int v0 = tile * TV;
  const SentTable tb = tabs[s];

  for (int c = tid; c < TV; c += SC_THREADS) {
    Lsh[c] = th0;
    Dsh[c] = 0.f;
  }
  if (tid < 2) s_lohi[tid] = lower_bound_tok(tb.entries + tb.uni_off, (int)tb.uni_cnt, v0 + tid * TV);
  __syncthreads();
  for (int e = s_lohi[0] + tid; e < s_lohi[1]; e += SC_THREADS) {
    const int2 en = tb.entries[tb.uni_off + e];
    Lsh[en.x - v0] = th0 + th1 * __int_as_float(en.y);
  }
  const float bias_e = eos_bias ? eos_bias[s] : 0.f;
  const float thn[3] = {th2, th3, th4};

  for (int k = 0; k < K; ++k) {
    const int row = s * K + k;
    Cand *out = topk + ((size_t)row * ntiles + tile) * K;
    __syncthreads();                                // Lsh/Dsh/s_lohi settled, buffers free
    if (q[row] == -INFINITY) {                      // dead slot: nothing to score
      if (tid == 0) stats[(size_t)row * ntiles + tile] = make_float2(-INFINITY, 0.f);
      if (tid < K) out[tid] = Cand{-INFINITY, -1};
      continue;
    }
    if (tid < 3) {
      const int off = ranges[row * 6 + tid * 2], cnt = ranges[row * 6 + tid * 2 + 1];
      int lo = 0, hi = 0;
      if (cnt > 0 && off >= 0 && (int64_t)off + cnt <= (int64_t)tb.n_entries) {
        lo = off + lower_bound_tok(tb.entries + off, cnt, v0);
        hi = off + lower_bound_tok(tb.entries + off, cnt, v0 + TV);
      }
      s_lohi[2 + 2 * tid] = lo;
      s_lohi[3 + 2 * tid] = hi;
    }
    if (tid == 0) s_cnt = 0;
    __syncthreads();
    const bool sparse = s_lohi[3] > s_lohi[2] || s_lohi[5] > s_lohi[4] || s_lohi[7] > s_lohi[6];
    if (sparse) {
      // one order at a time: words are unique within an order
      for (int o = 0; o < 3; ++o) {
        for (int e = s_lohi[2 + 2 * o] + tid; e < s_lohi[3 + 2 * o]; e += SC_THREADS) {
          const int2 en = tb.entries[e];
          Dsh[en.x - v0] += thn[o] * __int_as_float(en.y);
        }
        __syncthreads();
      }
    }

    // one coalesced read of the row's logits in this tile
    float val[VPT];
    const float *rp = logits + (size_t)row * ld;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int c = v0 + 1024 * g + 4 * tid;
      float4 f = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      if (c < V) f = *(const float4 *)(rp + c);
      val[4 * g + 0] = f.x;
      val[4 * g + 1] = (c + 1 < V) ? f.y : -INFINITY;
      val[4 * g + 2] = (c + 2 < V) ? f.z : -INFINITY;
      val[4 * g + 3] = (c + 3 < V) ? f.w : -INFINITY;
    }
    if (eos >= v0 && eos < v0 + TV) {
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (v0 + 1024 * g + 4 * tid + e == eos) val[4 * g + e] += bias_e;
    }

    // log-softmax partials over the tile: (max, sum exp(x - max))
    float mt = -INFINITY;
#pragma unroll
    for (int i = 0; i < VPT; ++i) mt = fmaxf(mt, val[i]);
    float st = 0.f;
    if (mt != -INFINITY) {
#pragma unroll
      for (int i = 0; i < VPT; ++i) st += __expf(val[i] - mt);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float om = __shfl_xor(mt, off, 64), os = __shfl_xor(st, off, 64);
      lse_combine(mt, st, om, os);
    }

    // x = logit + lambda * L(h, y)
    float x[VPT];
    float mx = -INFINITY;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int cl = 1024 * g + 4 * tid;
      const float4 lb = *(const float4 *)(&Lsh[cl]);
      const float4 ld4 = *(const float4 *)(&Dsh[cl]);
      x[4 * g + 0] = val[4 * g + 0] + lam * (lb.x + ld4.x);
      x[4 * g + 1] = val[4 * g + 1] + lam * (lb.y + ld4.y);
      x[4 * g + 2] = val[4 * g + 2] + lam * (lb.z + ld4.z);
      x[4 * g + 3] = val[4 * g + 3] + lam * (lb.w + ld4.w);
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) mx = fmaxf(mx, x[i]);

    // threshold: the K-th largest lane maximum of a wave bounds the tile's
    // K-th largest value from below
    float tau = -INFINITY;
    {
      float v = mx;
      for (int r = 0; r < K; ++r) {
        const float m = wave_max(v);
        tau = m;
        if (m == -INFINITY) break;
        const unsigned long long bal = __ballot(v == m);
        const int first = __ffsll((long long)bal) - 1;
        if (lane == first) v = -INFINITY;
      }
    }
    if (lane == 0) {
      s_rf[wid] = mt;
      s_rs[wid] = st;
      s_rf[4 + wid] = tau;
    }
    __syncthreads();
    if (tid == 0) {
      float m = s_rf[0], sm = s_rs[0];
      for (int w = 1; w < SC_THREADS / 64; ++w) lse_combine(m, sm, s_rf[w], s_rs[w]);
      stats[(size_t)row * ntiles + tile] = make_float2(m, sm);
    }
    tau = fmaxf(fmaxf(s_rf[4], s_rf[5]), fmaxf(s_rf[6], s_rf[7]));

    bool fallback = (tau == -INFINITY);
    if (!fallback) {
#pragma unroll
      for (int i = 0; i < VPT; ++i) {
        if (x[i] >= tau && x[i] != -INFINITY) {
          const int pos = atomicAdd(&s_cnt, 1);
          if (pos < SC_CAP) {
            cx[pos] = x[i];
            cv[pos] = v0 + 1024 * (i >> 2) + 4 * tid + (i & 3);
          }
        }
      }
      __syncthreads();
      fallback = s_cnt > SC_CAP;
    }
    if (!fallback) {
      // one wave selects the K best of the compacted candidates
      if (wid == 0) {
        const int n = s_cnt;
        unsigned taken = 0;
        for (int r = 0; r < K; ++r) {
          float bx = -INFINITY;
          int bv = 0x7FFFFFFF, bj = -1;
          for (int jj = 0, j = lane; j < n; ++jj, j += 64) {
            if (taken & (1u << jj)) continue;
            if (better(cx[j], cv[j], bx, bv)) { bx = cx[j]; bv = cv[j]; bj = jj; }
          }
          float wx = bx;
          int wv = bv;
          wave_argmax(wx, wv);
          if (bj >= 0 && bv == wv) taken |= 1u << bj;
          if (lane == 0) out[r] = (wv == 0x7FFFFFFF) ? Cand{-INFINITY, -1} : Cand{wx, wv};
        }
      }
    } else {
      // exact block-wide selection straight from the registers (ties or very
      // few valid columns)
      unsigned taken = 0;
      for (int r = 0; r < K; ++r) {
        float bx = -INFINITY;
        int bv = 0x7FFFFFFF, bi = -1;
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
          const int c = v0 + 1024 * (i >> 2) + 4 * tid + (i & 3);
          if (!(taken & (1u << i)) && c < V && better(x[i], c, bx, bv)) {
            bx = x[i];
            bv = c;
            bi = i;
          }
        }
        float wx = bx;
        int wv = bv;
        wave_argmax(wx, wv);
        __syncthreads();
        if (lane == 0) {
          s_rf[wid] = wx;
          s_ri[wid] = wv;
        }
        __syncthreads();
        float gx = s_rf[0];
        int gv = s_ri[0];
        for (int w = 1; w < SC_THREADS / 64; ++w)
          if (better(s_rf[w], s_ri[w], gx, gv)) { gx = s_rf[w]; gv = s_ri[w]; }
        if (bi >= 0 && bv == gv) taken |= 1u << bi;
        if (tid == 0) out[r] = (gv == 0x7FFFFFFF) ? Cand{-INFINITY, -1} : Cand{gx, gv};
      }
    }
    if (sparse) {
      __syncthreads();
      for (int o = 0; o < 3; ++o)
        for (int e = s_lohi[2 + 2 * o] + tid; e < s_lohi[3 + 2 * o]; e += SC_THREADS)
          Dsh[tb.entries[e].x - v0] = 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// Merge/select (TopB per sentence), EOS handling, realignment, context probes
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256)
void k_merge(int V, int K, int ntiles, int eos, int t_idx, int M,
             const float2 *__restrict__ stats, const Cand *__restrict__ topk,
             double *__restrict__ q, uint64_t *__restrict__ ctx, uint64_t *__restrict__ hh,
             int *__restrict__ len, int *__restrict__ ranges, int *__restrict__ bp,
             int *__restrict__ tok, double *__restrict__ qhist,
             const SentTable *__restrict__ tabs, int *__restrict__ parent_out,
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

  const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  if (tid < K) {
    const int row = s * K + tid;
    s_q[tid] = q[row];
    s_ctx[tid] = ctx[row];
    s_hh[tid] = hh[row];
    s_len[tid] = len[row];
  }
  __syncthreads();

  // each row: log-sum-exp over the tiles, and its K best by merging the
  // per-tile sorted lists (one list head per lane)
  for (int k = wid; k < K; k += 4) {
    const int row = s * K + k;
    if (s_q[k] == -INFINITY) {
      if (lane < K) {
        s_rx[k][lane] = -INFINITY;
        s_rv[k][lane] = -1;
      }
      if (lane == 0) s_lse[k] = 0.0;
      continue;
    }
    const float2 st = lane < ntiles ? stats[(size_t)row * ntiles + lane] : make_float2(-INFINITY, 0.f);
    double m = (double)st.x;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmax(m, __shfl_xor(m, off, 64));
    double part = (st.x != -INFINITY) ? (double)st.y * exp((double)st.x - m) : 0.0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
    if (lane == 0) s_lse[k] = m + log(part);

    int p = 0;
    const Cand *lst = topk + ((size_t)row * ntiles + lane) * K;
    for (int r = 0; r < K; ++r) {
      float hx = -INFINITY;
      int hv = 0x7FFFFFFF;
      if (lane < ntiles && p < K) {
        const Cand c = lst[p];
        if (c.v >= 0) { hx = c.x; hv = c.v; }
      }
      float wx = hx;
      int wv = hv;
      wave_argmax(wx, wv);
      if (lane < ntiles && hv == wv && wv != 0x7FFFFFFF) ++p;
      if (lane == 0) {
        s_rx[k][r] = wx;
        s_rv[k][r] = (wv == 0x7FFFFFFF) ? -1 : wv;
      }
    }
  }
  __syncthreads();

  if (tid < K) {                                    // defaults for any slot left unset
    s_selk[tid] = 0;
    s_selv[tid] = 0;
    s_sels[tid] = -INFINITY;
  }
  __syncthreads();
  // TopB over the sentence: score = q_k + (x - lse_k) in fp64, ties by k*V + v
  if (wid == 0) {
    int p = 0, nsel = 0;
    for (int r = 0; r < K; ++r) {
      double sc = -INFINITY;
      long long flat = 0x7FFFFFFFFFFFFFFFll;
      if (lane < K && p < K && s_rv[lane][p] >= 0 && s_q[lane] != -INFINITY) {
        sc = s_q[lane] + ((double)s_rx[lane][p] - s_lse[lane]);
        flat = (long long)lane * V + s_rv[lane][p];
      }
      double wsc = sc;
      long long wfl = flat;
      wave_argmax_d(wsc, wfl);
      if (wsc == -INFINITY || wfl == 0x7FFFFFFFFFFFFFFFll) break;
      if (lane < K && flat == wfl) ++p;
      if (lane == 0) {
        s_selk[r] = (int)(wfl / V);
        s_selv[r] = (int)(wfl % V);
        s_sels[r] = wsc;
      }
      ++nsel;
    }
    // fewer finite candidates than slots: the remaining slots take the -inf
    // candidates (every column of the dead rows) in flat-index order
    if (lane == 0) {
      int r = nsel;
      for (int k = 0; k < K && r < K; ++k) {
        if (s_q[k] != -INFINITY) continue;
        for (int v = 0; v < V && r < K; ++v, ++r) {
          s_selk[r] = k;
          s_selv[r] = v;
          s_sels[r] = -INFINITY;
        }
      }
    }
  }
  __syncthreads();

  if (tid < K) {
    const int j = tid, k = s_selk[j], v = s_selv[j];
    const double sc = s_sels[j];
    const int row = s * K + j;
    const size_t hidx = (size_t)t_idx * M + row;
    bp[hidx] = k;
    tok[hidx] = v;
    qhist[hidx] = sc;
    if (parent_out) parent_out[row] = k;
    if (token_out) token_out[row] = v;
    if (score_out) score_out[row] = sc;
    const bool live = sc != -INFINITY && v != eos;   // EOS: pushed to F (qhist), then masked
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
  if (tid < 3 * K) {
    const int j = tid / 3, o = tid % 3;
    int2 r = make_int2(0, 0);
    if (s_live[j] && s_nlen[j] >= o + 1) r = probe(tabs[s], s_nctx[j] & ((1ull << (21 * (o + 1))) - 1));
    const int row = s * K + j;
    ranges[row * 6 + o * 2] = r.x;
    ranges[row * 6 + o * 2 + 1] = r.y;
  }
}

// ---------------------------------------------------------------------------
// GetBestHypothesis: best F entry per sentence, traced back through bp/tok
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64)
void k_traceback(int K, int M, int T_max, int tcur, int eos, const double *__restrict__ q,
                 const int *__restrict__ bp, const int *__restrict__ tok,
                 const double *__restrict__ qhist, int *__restrict__ tokens_out,
                 int *__restrict__ len_out, double *__restrict__ score_out,
                 int *__restrict__ step_out, int *__restrict__ slot_out) {
  const int s = blockIdx.x, lane = threadIdx.x;
  double bs = -INFINITY;
  long long bkey = 0x7FFFFFFFFFFFFFFFll;   // t * K + j: earlier step, then lower slot
  for (int i = lane; i < tcur * K; i += 64) {
    const int t = i / K, j = i % K;
    const size_t idx = (size_t)t * M + s * K + j;
    const double sc = qhist[idx];
    if (tok[idx] == eos && sc != -INFINITY && better_d(sc, i, bs, bkey)) { bs = sc; bkey = i; }
  }
  if (tcur > 0) {
    for (int j = lane; j < K; j += 64) {
      const double sc = q[s * K + j];
      const long long key = (long long)(tcur - 1) * K + j;
      if (sc != -INFINITY && better_d(sc, key, bs, bkey)) { bs = sc; bkey = key; }
    }
  }
  wave_argmax_d(bs, bkey);
  const int found = bs != -INFINITY;
  const int bt = found ? (int)(bkey / K) : -1;
  for (int tt = lane; tt < T_max; tt += 64)
    if (tt > bt) tokens_out[(size_t)s * T_max + tt] = -1;
  if (lane == 0) {
    int j = found ? (int)(bkey % K) : -1;
    if (slot_out) slot_out[s] = j;
    if (step_out) step_out[s] = bt;
    len_out[s] = bt + 1;
    score_out[s] = bs;
    for (int tt = bt; tt >= 0; --tt) {
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
  const int64_t n = (int64_t)M * H;
  const int threads = 256;
  hipLaunchKernelGGL(k_synth_hidden, dim3((unsigned)((n + threads - 1) / threads)), dim3(threads), 0, st,
                     hh, hidden, M, H);
  return hipGetLastError();
}

hipError_t launch_state_init(int B, int K, uint64_t seed, double *q, uint64_t *ctx, uint64_t *hh,
                             int *len, int *ranges, hipStream_t st) {
  const int n = B * K;
  hipLaunchKernelGGL(k_state_init, dim3((n + 255) / 256), dim3(256), 0, st, B, K, seed, q, ctx, hh, len,
                     ranges);
  return hipGetLastError();
}

hipError_t launch_state_probe(int B, int K, const SentTable *tabs, const double *q, const uint64_t *ctx,
                              const int *len, int *ranges, hipStream_t st) {
  const int n = B * K * 3;
  hipLaunchKernelGGL(k_state_probe, dim3((n + 255) / 256), dim3(256), 0, st, B, K, tabs, q, ctx, len,
                     ranges);
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
  p.remap = ((p.nMb * p.nNb) % 8 == 0) ? 1 : 0;
  return p;
}

hipError_t launch_gemm(const uint16_t *A, const uint16_t *Bw, const float *bias, float *C, int M, int N,
                       int Kd, int64_t ldc, hipStream_t st) {
  const GemmPlan p = gemm_plan(M, N);
  const dim3 grid((unsigned)(p.nMb * p.nNb));
  if (p.bm == 256) {
    hipLaunchKernelGGL((k_gemm<256, 256, 128, 64>), grid, dim3(512), 0, st, A, Bw, bias, C, M, N, Kd, ldc,
                       p.nMb, p.nNb, p.remap);
  } else if (p.bm == 128) {
    hipLaunchKernelGGL((k_gemm<128, 128, 64, 64>), grid, dim3(256), 0, st, A, Bw, bias, C, M, N, Kd, ldc,
                       p.nMb, p.nNb, p.remap);
  } else {
    hipLaunchKernelGGL((k_gemm<64, 128, 32, 64>), grid, dim3(256), 0, st, A, Bw, bias, C, M, N, Kd, ldc,
                       p.nMb, p.nNb, p.remap);
  }
  return hipGetLastError();
}

ScorePlan score_plan(int B, int V) {
  ScorePlan p{};
  int vpt = 16;
  auto tiles = [&](int v) { return (V + 256 * v - 1) / (256 * v); };
  while (vpt > 4 && (int64_t)B * tiles(vpt) < 2048 && tiles(vpt / 2) <= LMBR_MAX_TILES) vpt /= 2;
  p.vpt = vpt;
  p.tv = 256 * vpt;
  p.ntiles = tiles(vpt);
  return p;
}

hipError_t launch_score(const ScorePlan &p, const float *logits, int64_t ld, int B, int V, int K,
                        const double *q, const int *ranges, const SentTable *tabs, const float *eos_bias,
                        int eos, float lam, const float *theta, float2 *stats, Cand *topk, hipStream_t st) {
  const dim3 grid((unsigned)p.ntiles, (unsigned)B);
#define LMBR_SCORE_ARGS                                                                                  \
  logits, ld, V, K, p.ntiles, q, ranges, tabs, eos_bias, eos, lam, theta[0], theta[1], theta[2], theta[3], \
      theta[4], stats, topk
  switch (p.vpt) {
    case 16: hipLaunchKernelGGL(k_score<16>, grid, dim3(SC_THREADS), 0, st, LMBR_SCORE_ARGS); break;
    case 8: hipLaunchKernelGGL(k_score<8>, grid, dim3(SC_THREADS), 0, st, LMBR_SCORE_ARGS); break;
    default: hipLaunchKernelGGL(k_score<4>, grid, dim3(SC_THREADS), 0, st, LMBR_SCORE_ARGS); break;
  }
#undef LMBR_SCORE_ARGS
  return hipGetLastError();
}

hipError_t launch_merge(int B, int V, int K, int ntiles, int eos, int t_idx, const float2 *stats,
                        const Cand *topk, double *q, uint64_t *ctx, uint64_t *hh, int *len, int *ranges,
                        int *bp, int *tok, double *qhist, const SentTable *tabs, int *parent_out,
                        int *token_out, double *score_out, hipStream_t st) {
  hipLaunchKernelGGL(k_merge, dim3(B), dim3(256), 0, st, V, K, ntiles, eos, t_idx, B * K, stats, topk, q,
                     ctx, hh, len, ranges, bp, tok, qhist, tabs, parent_out, token_out, score_out);
  return hipGetLastError();
}

hipError_t launch_traceback(int B, int K, int T_max, int tcur, int eos, const double *q, const int *bp,
                            const int *tok, const double *qhist, int *tokens_out, int *len_out,
                            double *score_out, int *step_out, int *slot_out, hipStream_t st) {
  hipLaunchKernelGGL(k_traceback, dim3(B), dim3(64), 0, st, K, B * K, T_max, tcur, eos, q, bp, tok, qhist,
                     tokens_out, len_out, score_out, step_out, slot_out);
  return hipGetLastError();
}

}  // namespace lmbr
