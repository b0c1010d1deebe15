// Device data layouts and kernel launchers of the LMBR beam decoder.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "lmbr.h"

#define LMBR_KMAX 16            // = LMBR_MAX_K
#define LMBR_MAX_TILES 128      // V-tiles per row (two list heads per lane in the merge)
#define LMBR_MAX_NT 8           // 256-column tiles per score tile (2048 columns)
#define LMBR_DIR_MIN 16         // successor lists longer than this carry a per-256-column directory

namespace lmbr {

constexpr uint64_t kEmptyKeyDev = ~0ull;
constexpr uint64_t kCtxMaskDev = (1ull << 63) - 1;

// One hash slot: packed (n-1)-word history -> its successor list.
struct __attribute__((aligned(16))) Slot {
  unsigned long long key;
  unsigned off;
  unsigned cnt;
};

// Per-sentence table descriptor (device memory).
struct SentTable {
  const Slot *slots;        // [mask + 1]
  const int2 *entries;      // {word, float bits of the posterior}, sorted by word per history
  const uint32_t *uni_tile; // [ceil(V / 256) + 1]: first unigram entry of each 256-column tile (absolute index)
  const float *uni_dense;   // [ceil(V / 256) * 256]: lambda * (theta0 + theta1 * p(v)), the history-free part of L
  const float *dense;       // dense layout only (else null): lambda * L, one row of ceil(V / 256) * 256 per history
  const uint32_t *slot_row; // ... and each hash slot's row there (row 0: the empty history)
  uint32_t mask;            // capacity - 1
  uint32_t uni_off;         // successors of the empty history (unigrams)
  uint32_t uni_cnt;
  uint32_t n_entries;
};

// One partial top-K entry: x = logit + lambda * L, v = word (-1 = none).
struct Cand {
  float x;
  int v;
};

// The decode options of a step (all null / 0: plain Algorithm 1).
struct StepOpts {
  const uint32_t *allowed;  // [B, ceil(V / 32)] allowed-word bits of each sentence, or null
  const int *steps;         // [B] last step (1-based) of each sentence, or null
  float *eosx;              // [M] the EOS column of x per row (written by the score pass), or null
  lmbr_sentence_record *sent;  // [B] per-sentence record (best finished value, backup), or null
  int length_norm;          // rank finished hypotheses by score per word
  int backup;               // keep the best non-surviving EOS candidate; F holds EOS entries only
  int prune;                // early pruning against the best finished value
  double prune_width;
  int *err;                 // device fault bits (LMBR_DEV_*), or null
};

struct GemmPlan {
  int bm, bn, threads, nMb, nNb, nt, remap;   // nt: column tiles per workgroup
};
struct ScorePlan {
  int ntiles;            // the score pass over logits: 1024-column tiles ...
  int score_nt;          // ... per strip (a workgroup per sentence and strip) ...
  int score_strips;      // ... and strips
  int fused_nt;          // the fused pass: 256-column tiles per strip (1 .. LMBR_MAX_NT) ...
  int fused_strips;      // ... and strips
};

GemmPlan gemm_plan(int M, int N);
ScorePlan score_plan(int B, int K, int V);

hipError_t launch_synth_hidden(const uint64_t *hh, uint16_t *hidden, int M, int H, hipStream_t st);
hipError_t launch_state_init(int B, int K, uint64_t seed, double *q, uint64_t *ctx, uint64_t *hh, int *len,
                             int *ranges, lmbr_sentence_record *sent, hipStream_t st);
hipError_t launch_state_probe(int B, int K, const SentTable *tabs, const double *q, const uint64_t *ctx,
                              const int *len, int *ranges, int *err, hipStream_t st);
hipError_t launch_transpose_bf16(const uint16_t *src, uint16_t *dst, int rows, int cols, hipStream_t st);
hipError_t launch_gather_rows(void *dst, const void *src, const int *rows, int n, int64_t row_bytes,
                              hipStream_t st);
// q: running scores [M] (device; only the live rows, finite score, are
// computed and stored, each to its own row of C; their number goes to
// *live_count when it is not null), or null for every row
hipError_t launch_gemm(const uint16_t *A, const uint16_t *Bw, const float *bias, float *C, int M, int N,
                       int Kd, int64_t ldc, const double *q, int *live_count, hipStream_t st);
hipError_t launch_add_scalar(float *x, size_t n, float c, hipStream_t st);
hipError_t launch_score(const ScorePlan &p, const float *logits, int64_t ld, int B, int V, int K,
                        const double *q, const int *ranges, const SentTable *tabs, const float *eos_bias,
                        int eos, float lam, const float *theta, const uint32_t *allowed, float *eosx,
                        float2 *stats, Cand *topk, int *err, hipStream_t st);
hipError_t launch_fused(const ScorePlan &p, const uint16_t *A, const uint16_t *Bw, const float *bias, int M,
                        int V, int Kd, int K, const int *ranges, const SentTable *tabs, const float *eos_bias,
                        int eos, float lam, const float *theta, const uint32_t *allowed, float *eosx,
                        const double *q, float2 *stats, Cand *topk, int *err, hipStream_t st);
hipError_t launch_merge(int B, int V, int K, int ntiles, int eos, int t_idx, const float2 *stats,
                        const Cand *topk, double *q, uint64_t *ctx, uint64_t *hh, int *len, int *ranges,
                        int *bp, int *tok, double *qhist, const SentTable *tabs, const StepOpts &opt,
                        int *parent_out, int *token_out, double *score_out, hipStream_t st);
hipError_t launch_traceback(int B, int K, int T_max, int tcur, int eos, const StepOpts &opt, const int *bp,
                            const int *tok, const double *qhist, int *tokens_out, int *len_out,
                            double *score_out, int *step_out, int *slot_out, hipStream_t st);

}  // namespace lmbr
