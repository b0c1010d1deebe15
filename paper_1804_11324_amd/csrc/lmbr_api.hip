// C ABI of the LMBR beam decoder: validation, the context and its device
// workspace, the posterior-table upload, and the per-step launch sequence.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "lmbr.h"
#include "tables.h"

using lmbr::Cand;
using lmbr::SentTable;
using lmbr::Slot;

struct lmbr_ctx {
  lmbr_config cfg{};
  int M = 0;
  lmbr::ScorePlan sp{};
  uint16_t *hidden = nullptr;      // [M, H] (built-in model)
  float2 *stats = nullptr;         // [M, part_strips]
  Cand *topk = nullptr;            // [M, part_strips, K]
  int part_strips = 0;             // strips the partials are sized for (both score passes)
  SentTable *d_tabs = nullptr;     // [B]
  std::vector<SentTable> h_tabs;   // host mirror of d_tabs
  std::vector<void *> tab_mem;     // per-sentence table allocation the context owns (nullptr: the shared
                                   // empty table, or caller-owned memory)
  std::vector<size_t> tab_bytes;
  void *empty_tab = nullptr;
  const uint16_t *W = nullptr;     // [V, H] bf16
  uint16_t *W_owned = nullptr;
  const float *bias = nullptr;
  float *logits_ws = nullptr;      // [M, ld_ws] fp32: the two-pass step's logits
  int *live_count = nullptr;       // live rows the last two-pass projection computed
  int64_t ld_ws = 0;
  int step_path = LMBR_STEP_TWO_PASS;
  int l_layout = LMBR_L_SPARSE;    // layout of tables loaded from now on
  bool scored = false;             // partials of a score call await lmbr_select
  int strips = 0;                  // ... over this many column strips
  // decode options
  int length_norm = 0;
  int finish = LMBR_FINISH_AT_T;
  int early_prune = 0;
  double prune_width = 0.0;
  int *steps = nullptr;            // [B] per-sentence last step (device)
  bool has_steps = false;
  const uint32_t *allowed = nullptr;  // [B, ceil(V / 32)] caller-owned, or null
  float *eosx = nullptr;           // [M] EOS column of x per row (backup stack)
  // lmbr_decode's loop of T steps, captured once into a HIP graph on a private
  // stream and replayed while everything baked into its launches is the same
  struct DecodeKey {
    int32_t T = -1, t0 = -1;
    lmbr_beam_state st{};
    const float *eos_bias = nullptr;
    const uint16_t *W = nullptr;
    const float *bias = nullptr;
    int step_path = -1, length_norm = 0, finish = 0, early_prune = 0;
    double prune_width = 0.0;
    bool has_steps = false;
    const uint32_t *allowed = nullptr;
  };
  hipStream_t cap_stream = nullptr;
  struct DecodeGraph {
    DecodeKey key{};
    hipGraphExec_t exec = nullptr;
    uint64_t last_use = 0;
  };
  static constexpr int kDecodeGraphs = 4;   // distinct loops kept (least recently used replaced)
  DecodeGraph graphs[kDecodeGraphs];
  uint64_t graph_clock = 0;

  void *ws = nullptr;               // the workspace (caller-owned unless ws_owned)
  bool ws_owned = false;
  int *dev_err = nullptr;          // device fault bits (LMBR_DEV_*)
  void *scratch = nullptr;         // device address of `scratch` on the context's device
  int32_t *tb_tok = nullptr;       // [B, T_max] lmbr_decode's traceback staging ...
  int32_t *tb_len = nullptr;       // [B]
  double *tb_score = nullptr;      // [B]
  size_t bytes = 0;                // device bytes in use besides the tables
  std::string err;
};

// Scratch of lmbr_beam_step_logits_static: the score pass's per-(row, strip)
// partials and the EOS column, for callers that cannot allocate.  One copy per
// GPU, held until the process ends; calls that overlap on one GPU share it.
static __device__ __align__(256) unsigned char scratch[LMBR_STATIC_SCRATCH_BYTES];

namespace {

thread_local std::string g_create_err;

constexpr int kLiveMapMaxRows = 1 << 14;     // beams whose projection lists its live rows
constexpr size_t kDenseMaxBytes = (size_t)2 << 30;   // a sentence's dense L

// Device address of `scratch` per device, taken once per device with that
// device current (host code must never pass the symbol itself to a kernel).
std::mutex g_scratch_mu;
std::vector<void *> g_scratch_ptr;

hipError_t scratch_address(int dev, void **out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize((size_t)dev + 1, nullptr);
  if (!g_scratch_ptr[(size_t)dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[(size_t)dev] = p;
  }
  *out = g_scratch_ptr[(size_t)dev];
  return hipSuccess;
}

int32_t fail(lmbr_ctx *ctx, int32_t code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (ctx) ctx->err = buf;
  else g_create_err = buf;
  return code;
}

int32_t hip_fail(lmbr_ctx *ctx, hipError_t e, const char *what) {
  return fail(ctx, LMBR_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define LMBR_HIP(ctx, call)                                   \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #call);  \
  } while (0)

bool bad_ptr(const void *p) { return p == nullptr; }

int32_t check_state(lmbr_ctx *ctx, const lmbr_beam_state *st) {
  if (!st) return fail(ctx, LMBR_E_INVALID, "state is NULL");
  if (!st->q || !st->ctx || !st->hhash || !st->len || !st->ranges || !st->bp || !st->tok || !st->qhist)
    return fail(ctx, LMBR_E_INVALID, "a state buffer is NULL");
  if (st->t < 0 || st->t > ctx->cfg.T_max)
    return fail(ctx, LMBR_E_INVALID, "state t=%d outside [0, T_max=%d]", st->t, ctx->cfg.T_max);
  if ((ctx->finish == LMBR_FINISH_EOS_BACKUP || ctx->early_prune) && !st->sent)
    return fail(ctx, LMBR_E_INVALID, "the backup stack and early pruning need st->sent");
  return LMBR_OK;
}

// Where a step's score pass leaves its results for the merge: the
// per-(row, strip) log-softmax partials and candidate lists, and the EOS
// column of x (read by the backup stack).  The context's workspace holds one
// set; lmbr_beam_step_logits_static uses the library's static scratch.
struct Partials {
  float2 *stats;
  Cand *topk;
  float *eosx;
};

Partials ws_partials(const lmbr_ctx *ctx) { return Partials{ctx->stats, ctx->topk, ctx->eosx}; }

// The decode options as the kernels take them.
lmbr::StepOpts step_opts(const lmbr_ctx *ctx, const lmbr_beam_state *st, float *eosx) {
  const bool backup = ctx->finish == LMBR_FINISH_EOS_BACKUP;
  return lmbr::StepOpts{ctx->allowed,    ctx->has_steps ? ctx->steps : nullptr,
                        backup ? eosx : nullptr, st->sent, ctx->length_norm, backup ? 1 : 0,
                        ctx->early_prune, ctx->prune_width, ctx->dev_err};
}

// The EOS column buffer the score pass fills (backup stack only).
float *eosx_out(const lmbr_ctx *ctx, const Partials &pt) {
  return ctx->finish == LMBR_FINISH_EOS_BACKUP ? pt.eosx : nullptr;
}

// Validation of a configuration, shared by lmbr_workspace_bytes and lmbr_create.
int32_t check_config(const lmbr_config *cfg) {
  if (!cfg) return fail(nullptr, LMBR_E_INVALID, "config is NULL");
  const lmbr_config &c = *cfg;
  if (c.B < 1) return fail(nullptr, LMBR_E_INVALID, "B=%d must be >= 1", c.B);
  if (c.K < 1 || c.K > LMBR_MAX_K) return fail(nullptr, LMBR_E_CAPACITY, "K=%d outside 1..%d", c.K, LMBR_MAX_K);
  if (c.V < 2 || c.V > LMBR_MAX_V) return fail(nullptr, LMBR_E_CAPACITY, "V=%d outside 2..%d", c.V, LMBR_MAX_V);
  if (c.H < 64 || c.H % 64 != 0) return fail(nullptr, LMBR_E_INVALID, "H=%d must be a positive multiple of 64", c.H);
  if (c.T_max < 1) return fail(nullptr, LMBR_E_INVALID, "T_max=%d must be >= 1", c.T_max);
  if (c.eos_id < 0 || c.eos_id >= c.V) return fail(nullptr, LMBR_E_INVALID, "eos_id=%d outside [0, V)", c.eos_id);
  if (!std::isfinite(c.lambda)) return fail(nullptr, LMBR_E_INVALID, "lambda is not finite");
  for (int i = 0; i < 5; ++i)
    if (!std::isfinite(c.theta[i])) return fail(nullptr, LMBR_E_INVALID, "theta[%d] is not finite", i);
  if (!(c.load_factor == 0.f || (c.load_factor > 0.f && c.load_factor <= 0.9f)))
    return fail(nullptr, LMBR_E_INVALID, "load_factor outside (0, 0.9]");
  const int64_t M = (int64_t)c.B * c.K;
  if (M > (1 << 24) || M * (int64_t)c.T_max > ((int64_t)1 << 31))
    return fail(nullptr, LMBR_E_CAPACITY, "B*K=%lld or B*K*T_max too large", (long long)M);
  const lmbr::ScorePlan sp = lmbr::score_plan(c.B, c.K, c.V);
  if (sp.score_strips > LMBR_MAX_TILES || sp.fused_strips > LMBR_MAX_TILES)
    return fail(nullptr, LMBR_E_CAPACITY, "V=%d needs more than %d score tiles", c.V, LMBR_MAX_TILES);
  return LMBR_OK;
}

// Byte offsets of the context's buffers in its workspace (each 256-aligned).
struct WsLayout {
  size_t hidden, stats, topk, tabs, steps, eosx, logits, live_count, err, tb_tok, tb_len, tb_score, empty,
      total;
  size_t empty_tile_bytes, empty_dense_bytes, empty_bytes;
  int part_strips;
};

WsLayout ws_layout(const lmbr_config &c) {
  WsLayout L{};
  const size_t M = (size_t)c.B * c.K;
  const lmbr::ScorePlan sp = lmbr::score_plan(c.B, c.K, c.V);
  // the partials of either score pass: one (max, sum) and K candidates per
  // row and strip, for the larger of the two strip counts
  L.part_strips = std::max(sp.score_strips, sp.fused_strips);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (std::max<size_t>(bytes, 1) + 255) / 256 * 256;
    return o;
  };
  L.hidden = take(sizeof(uint16_t) * M * c.H);
  L.stats = take(sizeof(float2) * M * L.part_strips);
  L.topk = take(sizeof(Cand) * M * L.part_strips * c.K);
  L.tabs = take(sizeof(SentTable) * c.B);
  L.steps = take(sizeof(int32_t) * c.B);
  L.eosx = take(sizeof(float) * M);
  L.logits = take(sizeof(float) * M * (size_t)((c.V + 63) / 64 * 64));
  L.live_count = take(sizeof(int32_t));
  L.err = take(sizeof(int32_t));
  L.tb_tok = take(sizeof(int32_t) * c.B * (size_t)c.T_max);
  L.tb_len = take(sizeof(int32_t) * c.B);
  L.tb_score = take(sizeof(double) * c.B);
  // the empty table every sentence starts with: two empty slots and no
  // entries, all-zero unigram bounds, the dense history-free row lambda * theta0
  const size_t nt256 = (size_t)((c.V + 255) / 256);
  L.empty_tile_bytes = (sizeof(uint32_t) * (nt256 + 1) + 255) / 256 * 256;
  L.empty_dense_bytes = sizeof(float) * nt256 * 256;
  L.empty_bytes = 256 + L.empty_tile_bytes + L.empty_dense_bytes;
  L.empty = take(L.empty_bytes);
  L.total = off;
  return L;
}

template <typename T>
int32_t dalloc(lmbr_ctx *ctx, T **p, size_t count, const char *what) {
  const size_t b = std::max<size_t>(1, count) * sizeof(T);
  hipError_t e = hipMalloc((void **)p, b);
  if (e != hipSuccess) return fail(ctx, LMBR_E_HIP, "hipMalloc(%s, %zu bytes): %s", what, b, hipGetErrorString(e));
  ctx->bytes += b;
  return LMBR_OK;
}

// The merge and the state update of one step, after a score pass has written
// its partials (over `strips` column strips) to pt.
int32_t merge_step(lmbr_ctx *ctx, lmbr_beam_state *st, const Partials &pt, int strips, int32_t *parent_out,
                   int32_t *token_out, double *score_out, hipStream_t stream) {
  const lmbr_config &c = ctx->cfg;
  hipError_t e = lmbr::launch_merge(c.B, c.V, c.K, strips, c.eos_id, st->t, pt.stats, pt.topk, st->q,
                                    st->ctx, st->hhash, st->len, st->ranges, st->bp, st->tok, st->qhist,
                                    ctx->d_tabs, step_opts(ctx, st, pt.eosx), parent_out, token_out, score_out,
                                    stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "merge kernel launch");
  ctx->scored = false;
  st->t += 1;
  return LMBR_OK;
}

// The score pass over logits in memory.
int32_t score_logits(lmbr_ctx *ctx, const lmbr_beam_state *st, const float *logits, int64_t ld,
                     const float *eos_bias, const Partials &pt, hipStream_t stream) {
  const lmbr_config &c = ctx->cfg;
  if (ctx->sp.score_strips > ctx->part_strips) return fail(ctx, LMBR_E_CAPACITY, "score strips exceed the partials");
  hipError_t e = lmbr::launch_score(ctx->sp, logits, ld, c.B, c.V, c.K, st->q, st->ranges, ctx->d_tabs,
                                    eos_bias, c.eos_id, c.lambda, c.theta, ctx->allowed, eosx_out(ctx, pt),
                                    pt.stats, pt.topk, ctx->dev_err, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "score kernel launch");
  ctx->scored = true;
  ctx->strips = ctx->sp.score_strips;
  return LMBR_OK;
}

// The fused projection + score pass from decoder states (the logits never
// reach memory).
int32_t score_hidden(lmbr_ctx *ctx, const lmbr_beam_state *st, const uint16_t *hidden, const float *eos_bias,
                     hipStream_t stream) {
  const lmbr_config &c = ctx->cfg;
  if (ctx->sp.fused_strips > ctx->part_strips) return fail(ctx, LMBR_E_CAPACITY, "fused strips exceed the partials");
  hipError_t e = lmbr::launch_fused(ctx->sp, hidden, ctx->W, ctx->bias, ctx->M, c.V, c.H, c.K, st->ranges,
                                    ctx->d_tabs, eos_bias, c.eos_id, c.lambda, c.theta, ctx->allowed,
                                    eosx_out(ctx, ws_partials(ctx)), st->q, ctx->stats, ctx->topk, ctx->dev_err,
                                    stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "fused projection/score launch");
  ctx->scored = true;
  ctx->strips = ctx->sp.fused_strips;
  return LMBR_OK;
}

// The scoring half of a step from decoder states, by the context's step path:
// the projection into the logits workspace and the score pass over it, or the
// fused kernel.
int32_t score_step(lmbr_ctx *ctx, const lmbr_beam_state *st, const uint16_t *hidden, const float *eos_bias,
                   hipStream_t stream) {
  if (ctx->step_path == LMBR_STEP_FUSED) return score_hidden(ctx, st, hidden, eos_bias, stream);
  const lmbr_config &c = ctx->cfg;
  // only the live rows are projected (the score pass reads no dead row): each
  // workgroup of the projection lists the beam's live rows and takes its
  // block of them; row blocks past them exit at once (beams beyond
  // kLiveMapMaxRows rows, where every workgroup's listing would cost more than
  // it saves, are projected whole)
  const bool compact = ctx->M <= kLiveMapMaxRows;
  hipError_t e = lmbr::launch_gemm(hidden, ctx->W, ctx->bias, ctx->logits_ws, ctx->M, c.V, c.H, ctx->ld_ws,
                                   compact ? st->q : nullptr, compact ? ctx->live_count : nullptr, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "gemm launch");
  return score_logits(ctx, st, ctx->logits_ws, ctx->ld_ws, eos_bias, ws_partials(ctx), stream);
}

int32_t check_step(lmbr_ctx *ctx, const lmbr_beam_state *st) {
  int32_t rc = check_state(ctx, st);
  if (rc) return rc;
  if (st->t >= ctx->cfg.T_max) return fail(ctx, LMBR_E_STATE, "history full: t=%d == T_max", st->t);
  return LMBR_OK;
}

int32_t check_hidden(lmbr_ctx *ctx, const uint16_t *hidden) {
  if (!ctx->W) return fail(ctx, LMBR_E_STATE, "no projection set (lmbr_set_projection)");
  if (bad_ptr(hidden)) return fail(ctx, LMBR_E_INVALID, "hidden is NULL");
  if (((uintptr_t)hidden & 15) != 0) return fail(ctx, LMBR_E_INVALID, "hidden must be 16-byte aligned");
  return LMBR_OK;
}

int32_t check_logits(lmbr_ctx *ctx, const float *logits, int64_t ld) {
  if (bad_ptr(logits)) return fail(ctx, LMBR_E_INVALID, "logits is NULL");
  if (ld < ctx->cfg.V || ld % 4 != 0 || ((uintptr_t)logits & 15) != 0)
    return fail(ctx, LMBR_E_INVALID, "logits need ld >= V, ld %% 4 == 0 and 16-byte alignment");
  return LMBR_OK;
}

}  // namespace

extern "C" {

const char *lmbr_last_error(const lmbr_ctx *ctx) { return ctx ? ctx->err.c_str() : g_create_err.c_str(); }

size_t lmbr_workspace_bytes(const lmbr_config *cfg) {
  g_create_err.clear();
  if (check_config(cfg)) return 0;
  return ws_layout(*cfg).total;
}

int32_t lmbr_create(const lmbr_config *cfg, void *workspace, size_t bytes, lmbr_ctx **out) {
  g_create_err.clear();
  if (!cfg || !out) return fail(nullptr, LMBR_E_INVALID, "lmbr_create: NULL argument");
  *out = nullptr;
  int32_t rc = check_config(cfg);
  if (rc) return rc;
  const lmbr_config &c = *cfg;
  const WsLayout L = ws_layout(c);
  if (workspace && bytes < L.total)
    return fail(nullptr, LMBR_E_CAPACITY, "workspace of %zu bytes, %zu needed", bytes, L.total);
  if (((uintptr_t)workspace & 255) != 0) return fail(nullptr, LMBR_E_INVALID, "workspace must be 256-byte aligned");
  int dev_count = 0;
  hipError_t e = hipGetDeviceCount(&dev_count);
  if (e != hipSuccess || dev_count == 0)
    return fail(nullptr, LMBR_E_HIP, "no HIP device available (%s)", hipGetErrorString(e));

  int dev = 0;
  void *scr = nullptr;
  if ((e = hipGetDevice(&dev)) != hipSuccess || (e = scratch_address(dev, &scr)) != hipSuccess)
    return fail(nullptr, LMBR_E_HIP, "static scratch address: %s", hipGetErrorString(e));

  lmbr_ctx *ctx = new lmbr_ctx();
  ctx->cfg = c;
  ctx->scratch = scr;
  if (ctx->cfg.load_factor == 0.f) ctx->cfg.load_factor = 0.5f;
  ctx->M = c.B * c.K;
  ctx->sp = lmbr::score_plan(c.B, c.K, c.V);
  ctx->part_strips = L.part_strips;
  ctx->ld_ws = (c.V + 63) / 64 * 64;
  if (workspace) {
    ctx->ws = workspace;
  } else {
    e = hipMalloc(&ctx->ws, L.total);
    if (e != hipSuccess) {
      delete ctx;
      return fail(nullptr, LMBR_E_HIP, "hipMalloc(workspace, %zu bytes): %s", L.total, hipGetErrorString(e));
    }
    ctx->ws_owned = true;
  }
  ctx->bytes = L.total;
  char *w = (char *)ctx->ws;
  ctx->hidden = (uint16_t *)(w + L.hidden);
  ctx->stats = (float2 *)(w + L.stats);
  ctx->topk = (Cand *)(w + L.topk);
  ctx->d_tabs = (SentTable *)(w + L.tabs);
  ctx->steps = (int *)(w + L.steps);
  ctx->eosx = (float *)(w + L.eosx);
  ctx->logits_ws = (float *)(w + L.logits);
  ctx->live_count = (int *)(w + L.live_count);
  ctx->dev_err = (int *)(w + L.err);
  ctx->tb_tok = (int32_t *)(w + L.tb_tok);
  ctx->tb_len = (int32_t *)(w + L.tb_len);
  ctx->tb_score = (double *)(w + L.tb_score);
  ctx->empty_tab = w + L.empty;
  Slot empty[2];
  for (auto &sl : empty) sl = Slot{lmbr::kEmptyKey, 0u, 0u};
  const size_t nt256 = (size_t)((c.V + 255) / 256);
  std::vector<float> dense0(nt256 * 256, c.lambda * c.theta[0]);
  const int zero = 0;
  e = hipMemset(ctx->empty_tab, 0, L.empty_bytes);
  if (e == hipSuccess) e = hipMemcpy(ctx->empty_tab, empty, sizeof empty, hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy((char *)ctx->empty_tab + 256 + L.empty_tile_bytes, dense0.data(), L.empty_dense_bytes,
                  hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(ctx->dev_err, &zero, sizeof zero, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(ctx->live_count, &ctx->M, sizeof(int), hipMemcpyHostToDevice);
  ctx->h_tabs.assign(c.B, SentTable{(const Slot *)ctx->empty_tab,
                                    (const int2 *)((char *)ctx->empty_tab + sizeof empty),
                                    (const uint32_t *)((char *)ctx->empty_tab + 256),
                                    (const float *)((char *)ctx->empty_tab + 256 + L.empty_tile_bytes), nullptr,
                                    nullptr, 1u, 0u, 0u, 0u});
  ctx->tab_mem.assign(c.B, nullptr);
  ctx->tab_bytes.assign(c.B, 0);
  if (e == hipSuccess)
    e = hipMemcpy(ctx->d_tabs, ctx->h_tabs.data(), sizeof(SentTable) * c.B, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    hip_fail(ctx, e, "workspace set-up");
    g_create_err = ctx->err;
    lmbr_destroy(ctx);
    return LMBR_E_HIP;
  }
  *out = ctx;
  return LMBR_OK;
}

void lmbr_destroy(lmbr_ctx *ctx) {
  if (!ctx) return;
  (void)hipDeviceSynchronize();
  for (auto &g : ctx->graphs)
    if (g.exec) (void)hipGraphExecDestroy(g.exec);
  if (ctx->cap_stream) (void)hipStreamDestroy(ctx->cap_stream);
  for (void *p : ctx->tab_mem) if (p) (void)hipFree(p);
  if (ctx->ws_owned) (void)hipFree(ctx->ws);
  (void)hipFree(ctx->W_owned);
  delete ctx;
}

int32_t lmbr_device_status(lmbr_ctx *ctx, int32_t *bits, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (bits) *bits = 0;
  int v = 0;
  const int zero = 0;
  LMBR_HIP(ctx, hipStreamSynchronize(stream));
  LMBR_HIP(ctx, hipMemcpy(&v, ctx->dev_err, sizeof v, hipMemcpyDeviceToHost));
  if (v == 0) return LMBR_OK;
  LMBR_HIP(ctx, hipMemcpy(ctx->dev_err, &zero, sizeof zero, hipMemcpyHostToDevice));
  if (bits) *bits = v;
  return fail(ctx, LMBR_E_DEVICE, "device fault flag 0x%x:%s%s", v,
              (v & LMBR_DEV_NONFINITE) ? " non-finite log-softmax normaliser or score" : "",
              (v & LMBR_DEV_TABLE) ? " posterior table probe or range out of bounds" : "");
}

size_t lmbr_device_bytes(const lmbr_ctx *ctx) {
  if (!ctx) return 0;
  size_t b = ctx->bytes;
  for (size_t x : ctx->tab_bytes) b += x;
  return b;
}

int32_t lmbr_set_projection(lmbr_ctx *ctx, const uint16_t *w, int32_t layout, const float *bias,
                            hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (bad_ptr(w)) return fail(ctx, LMBR_E_INVALID, "lmbr_set_projection: w is NULL");
  if (layout != 0 && layout != 1) return fail(ctx, LMBR_E_INVALID, "layout=%d must be 0 ([V,H]) or 1 ([H,V])", layout);
  if (((uintptr_t)w & 15) != 0) return fail(ctx, LMBR_E_INVALID, "w must be 16-byte aligned");
  const lmbr_config &c = ctx->cfg;
  if (layout == 0) {
    ctx->W = w;
  } else {
    if (!ctx->W_owned) {
      int32_t rc = dalloc(ctx, &ctx->W_owned, (size_t)c.V * c.H, "repacked W");
      if (rc) return rc;
    }
    hipError_t e = lmbr::launch_transpose_bf16(w, ctx->W_owned, c.H, c.V, stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "transpose launch");
    ctx->W = ctx->W_owned;
  }
  ctx->bias = bias;
  return LMBR_OK;
}

}  // extern "C"

namespace {

// One sentence's posterior table as built on the host, ready for upload.
struct HostTable {
  std::vector<Slot> hs;                 // hash slots
  std::vector<int2> he;                 // successor lists (with directories)
  std::vector<uint32_t> ht;             // unigram bounds per 256 columns
  std::vector<float> hd;                // dense history-free row of lambda * L
  std::vector<float> hL;                // dense layout: lambda * L per history (without lambda * theta0)
  std::vector<uint32_t> hrow;           // dense layout: each slot's row
  size_t slot_bytes = 0, entry_bytes = 0, tile_bytes = 0, dense_bytes = 0, L_bytes = 0, row_bytes = 0, total = 0;
  uint32_t n_slots = 0, uni_off = 0, uni_cnt = 0, n_dev = 0;
};

// The host half of lmbr_load_posteriors: the hash, the successor lists and
// their directories, the unigram bounds and the dense rows, and the device
// bytes they take.
int32_t build_table(lmbr_ctx *ctx, int64_t n, const int32_t *order, const int32_t *tokens, const float *post,
                    HostTable &T) {
  const lmbr_config &c = ctx->cfg;
  lmbr_table_image img;
  char msg[256];
  int32_t rc = lmbr_table_build(c.V, n, order, tokens, post, c.load_factor, &img, msg, sizeof msg);
  if (rc) return fail(ctx, rc, "%s", msg);
  if (img.n_slots > (int64_t)UINT32_MAX || img.n_entries > (int64_t)UINT32_MAX) {
    lmbr_table_free(&img);
    return fail(ctx, LMBR_E_CAPACITY, "table too large");
  }
  // Device layout: the successor lists in the image's order; a list of more
  // than LMBR_DIR_MIN successors is preceded by its directory over the
  // 256-column tiles (the first entry index with word >= 256 t for t = 0 ..
  // ceil(V / 256), packed two per int2), so that a pass over one tile touches
  // only that tile's successors.  The unigram list gets its bounds per 256
  // columns, and a dense copy (below).
  const int ndir = (c.V + 255) / 256;
  const int64_t D = (ndir + 2) / 2;
  struct ListRef {
    uint32_t off, cnt;
    int64_t slot;                       // -1: the unigram list
  };
  std::vector<ListRef> lists;
  for (int64_t i = 0; i < img.n_slots; ++i)
    if (img.slot_key[i] != lmbr::kEmptyKey) lists.push_back({img.slot_off[i], img.slot_cnt[i], i});
  if (img.uni_cnt) lists.push_back({img.uni_off, img.uni_cnt, -1});
  std::sort(lists.begin(), lists.end(), [](const ListRef &x, const ListRef &y) { return x.off < y.off; });
  T.hs.resize((size_t)img.n_slots);
  for (int64_t i = 0; i < img.n_slots; ++i) T.hs[(size_t)i] = Slot{img.slot_key[i], 0u, img.slot_cnt[i]};
  std::vector<int2> &he = T.he;
  he.reserve((size_t)img.n_entries + 64);
  uint32_t uni_off = 0;
  for (const ListRef &l : lists) {
    const bool dir = l.slot >= 0 && l.cnt > LMBR_DIR_MIN;
    const size_t dpos = he.size();
    if (dir) he.resize(he.size() + (size_t)D, int2{0, 0});
    const uint32_t start = (uint32_t)he.size();
    for (uint32_t k = 0; k < l.cnt; ++k) {
      int2 v;
      v.x = img.entry_tok[l.off + k];
      std::memcpy(&v.y, &img.entry_post[l.off + k], 4);
      he.push_back(v);
    }
    if (dir) {
      std::vector<uint32_t> d((size_t)D * 2, 0u);
      uint32_t k = 0;
      for (int t = 0; t <= ndir; ++t) {
        while (k < l.cnt && (int64_t)img.entry_tok[l.off + k] < (int64_t)t * 256) ++k;
        d[(size_t)t] = start + k;
      }
      std::memcpy(&he[dpos], d.data(), sizeof(uint32_t) * d.size());
    }
    if (l.slot >= 0) T.hs[(size_t)l.slot].off = start;
    else uni_off = start;
  }
  if (he.size() > (size_t)INT32_MAX) {
    lmbr_table_free(&img);
    return fail(ctx, LMBR_E_CAPACITY, "table too large");
  }
  T.n_dev = (uint32_t)he.size();
  if (he.empty()) he.push_back(int2{0, 0});
  const int nt256 = (c.V + 255) / 256;
  T.ht.resize((size_t)nt256 + 1);
  {
    uint32_t e = 0;
    for (int t = 0; t <= nt256; ++t) {
      while (e < img.uni_cnt && img.entry_tok[img.uni_off + e] < t * 256) ++e;
      T.ht[(size_t)t] = uni_off + e;
    }
  }
  // the history-free part of L as a dense row: lambda * (theta0 + theta1 * p)
  // for unigrams, lambda * theta0 elsewhere (padded to whole 256-column tiles)
  const float lth0 = c.lambda * c.theta[0], lth1 = c.lambda * c.theta[1];
  T.hd.assign((size_t)nt256 * 256, lth0);
  for (uint32_t k = 0; k < img.uni_cnt; ++k)
    T.hd[(size_t)img.entry_tok[img.uni_off + k]] = lth0 + lth1 * img.entry_post[img.uni_off + k];
  auto up256 = [](size_t b) { return (b + 255) / 256 * 256; };
  T.slot_bytes = up256(sizeof(Slot) * T.hs.size());
  T.entry_bytes = up256(sizeof(int2) * he.size());
  T.tile_bytes = up256(sizeof(uint32_t) * T.ht.size());
  T.dense_bytes = up256(sizeof(float) * T.hd.size());
  // the dense layout (Section 2's matrix L, one row per history): the sparse
  // part built here, lambda * theta0 added on the device after the upload
  if (ctx->l_layout == LMBR_L_DENSE) {
    const int64_t nrows = lmbr_table_history_count(&img) + 1;
    const size_t ldL = (size_t)nt256 * 256;
    if ((double)nrows * (double)ldL * sizeof(float) > (double)kDenseMaxBytes) {
      lmbr_table_free(&img);
      return fail(ctx, LMBR_E_CAPACITY, "dense L of %lld histories x %zu words exceeds %zu bytes", (long long)nrows,
                  ldL, (size_t)kDenseMaxBytes);
    }
    T.hL.resize((size_t)nrows * ldL);
    T.hrow.resize((size_t)img.n_slots);
    if (lmbr_table_dense(&img, c.V, (int64_t)ldL, c.lambda, c.theta, T.hL.data(), T.hrow.data()) != LMBR_OK) {
      lmbr_table_free(&img);
      return fail(ctx, LMBR_E_INVALID, "dense L build");
    }
    T.L_bytes = up256(sizeof(float) * T.hL.size());
    T.row_bytes = up256(sizeof(uint32_t) * T.hrow.size());
  }
  T.n_slots = (uint32_t)img.n_slots;
  T.uni_off = uni_off;
  T.uni_cnt = img.uni_cnt;
  T.total = T.slot_bytes + T.entry_bytes + T.tile_bytes + T.dense_bytes + T.L_bytes + T.row_bytes;
  lmbr_table_free(&img);
  return LMBR_OK;
}

// The device half: the table into mem (at least T.total bytes, 256-aligned),
// ordered after the work already on `stream`, then the sentence's descriptor.
// owned: the context frees mem when the sentence is loaded again or at destroy.
int32_t install_table(lmbr_ctx *ctx, int32_t sentence, const HostTable &T, void *mem, bool owned,
                      hipStream_t stream) {
  const lmbr_config &c = ctx->cfg;
  char *m = (char *)mem;
  char *dense_L = T.hL.empty() ? nullptr : m + T.slot_bytes + T.entry_bytes + T.tile_bytes + T.dense_bytes;
  SentTable d{(const Slot *)m, (const int2 *)(m + T.slot_bytes), (const uint32_t *)(m + T.slot_bytes + T.entry_bytes),
              (const float *)(m + T.slot_bytes + T.entry_bytes + T.tile_bytes), (const float *)dense_L,
              dense_L ? (const uint32_t *)(dense_L + T.L_bytes) : nullptr, T.n_slots - 1u, T.uni_off, T.uni_cnt,
              T.n_dev};
  // ordered after earlier work on the stream that may still read the old table
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = hipMemcpy(m, T.hs.data(), sizeof(Slot) * T.hs.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(m + T.slot_bytes, T.he.data(), sizeof(int2) * T.he.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(m + T.slot_bytes + T.entry_bytes, T.ht.data(), sizeof(uint32_t) * T.ht.size(),
                  hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(m + T.slot_bytes + T.entry_bytes + T.tile_bytes, T.hd.data(), sizeof(float) * T.hd.size(),
                  hipMemcpyHostToDevice);
  if (e == hipSuccess && dense_L) {
    e = hipMemcpy(dense_L, T.hL.data(), sizeof(float) * T.hL.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy(dense_L + T.L_bytes, T.hrow.data(), sizeof(uint32_t) * T.hrow.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = lmbr::launch_add_scalar((float *)dense_L, T.hL.size(), c.lambda * c.theta[0], stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
  }
  if (e == hipSuccess) e = hipMemcpy(ctx->d_tabs + sentence, &d, sizeof d, hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(ctx, e, "posterior table upload");
  if (ctx->tab_mem[sentence]) (void)hipFree(ctx->tab_mem[sentence]);
  ctx->tab_mem[sentence] = owned ? mem : nullptr;
  ctx->tab_bytes[sentence] = T.total;
  ctx->h_tabs[sentence] = d;
  return LMBR_OK;
}

}  // namespace

extern "C" {

int32_t lmbr_load_posteriors(lmbr_ctx *ctx, int32_t sentence, int64_t n, const int32_t *order,
                             const int32_t *tokens, const float *post, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (sentence < 0 || sentence >= ctx->cfg.B)
    return fail(ctx, LMBR_E_INVALID, "sentence=%d outside [0, B=%d)", sentence, ctx->cfg.B);
  HostTable T;
  int32_t rc = build_table(ctx, n, order, tokens, post, T);
  if (rc) return rc;
  void *mem = nullptr;
  hipError_t e = hipMalloc(&mem, T.total);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMalloc(posterior table)");
  rc = install_table(ctx, sentence, T, mem, true, stream);
  if (rc) (void)hipFree(mem);
  return rc;
}

size_t lmbr_table_bytes(lmbr_ctx *ctx, int64_t n, const int32_t *order, const int32_t *tokens, const float *post) {
  if (!ctx) return 0;
  HostTable T;
  if (build_table(ctx, n, order, tokens, post, T) != LMBR_OK) return 0;
  return T.total;
}

int32_t lmbr_load_posteriors_into(lmbr_ctx *ctx, int32_t sentence, int64_t n, const int32_t *order,
                                  const int32_t *tokens, const float *post, void *table_mem, size_t bytes,
                                  hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (sentence < 0 || sentence >= ctx->cfg.B)
    return fail(ctx, LMBR_E_INVALID, "sentence=%d outside [0, B=%d)", sentence, ctx->cfg.B);
  if (!table_mem || ((uintptr_t)table_mem & 255) != 0)
    return fail(ctx, LMBR_E_INVALID, "table memory must be non-NULL and 256-byte aligned");
  HostTable T;
  int32_t rc = build_table(ctx, n, order, tokens, post, T);
  if (rc) return rc;
  if (bytes < T.total)
    return fail(ctx, LMBR_E_CAPACITY, "table memory of %zu bytes, %zu needed", bytes, T.total);
  return install_table(ctx, sentence, T, table_mem, false, stream);
}

int32_t lmbr_state_init(lmbr_ctx *ctx, lmbr_beam_state *st, uint64_t seed, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (st) st->t = 0;
  int32_t rc = check_state(ctx, st);
  if (rc) return rc;
  hipError_t e = lmbr::launch_state_init(ctx->cfg.B, ctx->cfg.K, seed, st->q, st->ctx, st->hhash, st->len,
                                         st->ranges, st->sent, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "state init launch");
  return LMBR_OK;
}

int32_t lmbr_state_probe(lmbr_ctx *ctx, lmbr_beam_state *st, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_state(ctx, st);
  if (rc) return rc;
  hipError_t e = lmbr::launch_state_probe(ctx->cfg.B, ctx->cfg.K, ctx->d_tabs, st->q, st->ctx, st->len,
                                          st->ranges, ctx->dev_err, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "state probe launch");
  return LMBR_OK;
}

int32_t lmbr_synth_hidden(lmbr_ctx *ctx, const lmbr_beam_state *st, uint16_t *hidden, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_state(ctx, st);
  if (rc) return rc;
  if (bad_ptr(hidden)) return fail(ctx, LMBR_E_INVALID, "hidden is NULL");
  hipError_t e = lmbr::launch_synth_hidden(st->hhash, hidden, ctx->M, ctx->cfg.H, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "synth launch");
  return LMBR_OK;
}

int32_t lmbr_project(lmbr_ctx *ctx, const uint16_t *hidden, float *logits, int64_t ld, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (!ctx->W) return fail(ctx, LMBR_E_STATE, "no projection set (lmbr_set_projection)");
  if (bad_ptr(hidden) || bad_ptr(logits)) return fail(ctx, LMBR_E_INVALID, "hidden or logits is NULL");
  if (((uintptr_t)hidden & 15) != 0) return fail(ctx, LMBR_E_INVALID, "hidden must be 16-byte aligned");
  if (ld < ctx->cfg.V) return fail(ctx, LMBR_E_INVALID, "ld=%lld < V=%d", (long long)ld, ctx->cfg.V);
  hipError_t e = lmbr::launch_gemm(hidden, ctx->W, ctx->bias, logits, ctx->M, ctx->cfg.V, ctx->cfg.H, ld, nullptr,
                                   nullptr, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "gemm launch");
  return LMBR_OK;
}

int32_t lmbr_beam_step(lmbr_ctx *ctx, lmbr_beam_state *st, const uint16_t *hidden, const float *eos_bias,
                       int32_t *parent_out, int32_t *token_out, double *score_out, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_step(ctx, st);
  if (rc || (rc = check_hidden(ctx, hidden))) return rc;
  if ((rc = score_step(ctx, st, hidden, eos_bias, stream))) return rc;
  return merge_step(ctx, st, ws_partials(ctx), ctx->strips, parent_out, token_out, score_out, stream);
}

int32_t lmbr_beam_step_logits(lmbr_ctx *ctx, lmbr_beam_state *st, const float *logits, int64_t ld,
                              const float *eos_bias, int32_t *parent_out, int32_t *token_out,
                              double *score_out, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_step(ctx, st);
  if (rc || (rc = check_logits(ctx, logits, ld))) return rc;
  if ((rc = score_logits(ctx, st, logits, ld, eos_bias, ws_partials(ctx), stream))) return rc;
  return merge_step(ctx, st, ws_partials(ctx), ctx->strips, parent_out, token_out, score_out, stream);
}

size_t lmbr_static_scratch_bytes(const lmbr_config *cfg) {
  g_create_err.clear();
  if (check_config(cfg)) return 0;
  const lmbr::ScorePlan sp = lmbr::score_plan(cfg->B, cfg->K, cfg->V);
  const size_t M = (size_t)cfg->B * cfg->K, n = M * (size_t)sp.score_strips;
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  return up(sizeof(float2) * n) + up(sizeof(Cand) * n * cfg->K) + up(sizeof(float) * M);
}

int32_t lmbr_beam_step_logits_static(lmbr_ctx *ctx, lmbr_beam_state *st, const float *logits, int64_t ld,
                                     const float *eos_bias, int32_t *parent_out, int32_t *token_out,
                                     double *score_out, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_step(ctx, st);
  if (rc || (rc = check_logits(ctx, logits, ld))) return rc;
  const size_t need = lmbr_static_scratch_bytes(&ctx->cfg);
  if (need > LMBR_STATIC_SCRATCH_BYTES)
    return fail(ctx, LMBR_E_CAPACITY, "the step needs %zu bytes of scratch, the static scratch holds %u", need,
                (unsigned)LMBR_STATIC_SCRATCH_BYTES);
  // every (row, strip) partial and every live row's EOS column is written by
  // the score pass before the merge reads it: nothing needs clearing
  const size_t M = (size_t)ctx->M, n = M * (size_t)ctx->sp.score_strips;
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  char *base = (char *)ctx->scratch;
  const Partials pt{(float2 *)base, (Cand *)(base + up(sizeof(float2) * n)),
                    (float *)(base + up(sizeof(float2) * n) + up(sizeof(Cand) * n * ctx->cfg.K))};
  if ((rc = score_logits(ctx, st, logits, ld, eos_bias, pt, stream))) return rc;
  return merge_step(ctx, st, pt, ctx->sp.score_strips, parent_out, token_out, score_out, stream);
}

int32_t lmbr_score(lmbr_ctx *ctx, const lmbr_beam_state *st, const uint16_t *hidden, const float *eos_bias,
                   hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_step(ctx, st);
  if (rc || (rc = check_hidden(ctx, hidden))) return rc;
  return score_step(ctx, st, hidden, eos_bias, stream);
}

int32_t lmbr_score_logits(lmbr_ctx *ctx, const lmbr_beam_state *st, const float *logits, int64_t ld,
                          const float *eos_bias, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_step(ctx, st);
  if (rc || (rc = check_logits(ctx, logits, ld))) return rc;
  return score_logits(ctx, st, logits, ld, eos_bias, ws_partials(ctx), stream);
}

int32_t lmbr_select(lmbr_ctx *ctx, lmbr_beam_state *st, int32_t *parent_out, int32_t *token_out,
                    double *score_out, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_step(ctx, st);
  if (rc) return rc;
  if (!ctx->scored) return fail(ctx, LMBR_E_STATE, "lmbr_select without a preceding score call");
  return merge_step(ctx, st, ws_partials(ctx), ctx->strips, parent_out, token_out, score_out, stream);
}

int32_t lmbr_projected_rows(lmbr_ctx *ctx, int32_t *rows, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  if (!rows) return fail(ctx, LMBR_E_INVALID, "rows is NULL");
  LMBR_HIP(ctx, hipStreamSynchronize(stream));
  int v = ctx->M;
  if (ctx->step_path == LMBR_STEP_TWO_PASS && ctx->M <= kLiveMapMaxRows)
    LMBR_HIP(ctx, hipMemcpy(&v, ctx->live_count, sizeof v, hipMemcpyDeviceToHost));
  *rows = v;
  return LMBR_OK;
}

int32_t lmbr_set_lmbr_layout(lmbr_ctx *ctx, int32_t layout) {
  if (!ctx) return LMBR_E_INVALID;
  if (layout != LMBR_L_SPARSE && layout != LMBR_L_DENSE)
    return fail(ctx, LMBR_E_INVALID, "layout %d must be LMBR_L_SPARSE or LMBR_L_DENSE", layout);
  ctx->l_layout = layout;
  return LMBR_OK;
}

int32_t lmbr_set_step_path(lmbr_ctx *ctx, int32_t path) {
  if (!ctx) return LMBR_E_INVALID;
  if (path != LMBR_STEP_TWO_PASS && path != LMBR_STEP_FUSED)
    return fail(ctx, LMBR_E_INVALID, "step path %d must be LMBR_STEP_TWO_PASS or LMBR_STEP_FUSED", path);
  ctx->step_path = path;
  return LMBR_OK;
}

int32_t lmbr_set_decode_options(lmbr_ctx *ctx, const lmbr_decode_options *opt) {
  if (!ctx) return LMBR_E_INVALID;
  if (!opt) return fail(ctx, LMBR_E_INVALID, "lmbr_set_decode_options: opt is NULL");
  if (opt->length_norm != 0 && opt->length_norm != 1)
    return fail(ctx, LMBR_E_INVALID, "length_norm=%d must be 0 or 1", opt->length_norm);
  if (opt->finish != LMBR_FINISH_AT_T && opt->finish != LMBR_FINISH_EOS_BACKUP)
    return fail(ctx, LMBR_E_INVALID, "finish=%d is not an LMBR_FINISH_* value", opt->finish);
  if (opt->early_prune != 0 && opt->early_prune != 1)
    return fail(ctx, LMBR_E_INVALID, "early_prune=%d must be 0 or 1", opt->early_prune);
  if (opt->early_prune && !(opt->prune_width >= 0.0))
    return fail(ctx, LMBR_E_INVALID, "prune_width must be >= 0");
  ctx->length_norm = opt->length_norm;
  ctx->finish = opt->finish;
  ctx->early_prune = opt->early_prune;
  ctx->prune_width = opt->early_prune ? opt->prune_width : 0.0;
  return LMBR_OK;
}

int32_t lmbr_set_sentence_steps(lmbr_ctx *ctx, const int32_t *steps) {
  if (!ctx) return LMBR_E_INVALID;
  if (!steps) {
    ctx->has_steps = false;
    return LMBR_OK;
  }
  for (int s = 0; s < ctx->cfg.B; ++s)
    if (steps[s] < 1 || steps[s] > ctx->cfg.T_max)
      return fail(ctx, LMBR_E_INVALID, "steps[%d]=%d outside [1, T_max=%d]", s, steps[s], ctx->cfg.T_max);
  LMBR_HIP(ctx, hipDeviceSynchronize());            // no step in flight reads the old values
  LMBR_HIP(ctx, hipMemcpy(ctx->steps, steps, sizeof(int32_t) * ctx->cfg.B, hipMemcpyHostToDevice));
  ctx->has_steps = true;
  return LMBR_OK;
}

int32_t lmbr_set_constraints(lmbr_ctx *ctx, const uint32_t *allowed) {
  if (!ctx) return LMBR_E_INVALID;
  if (((uintptr_t)allowed & 3) != 0) return fail(ctx, LMBR_E_INVALID, "allowed must be 4-byte aligned");
  ctx->allowed = allowed;
  return LMBR_OK;
}

int32_t lmbr_traceback(lmbr_ctx *ctx, const lmbr_beam_state *st, int32_t *tokens_out, int32_t *len_out,
                       double *score_out, int32_t *step_out, int32_t *slot_out, hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_state(ctx, st);
  if (rc) return rc;
  if (bad_ptr(tokens_out) || bad_ptr(len_out) || bad_ptr(score_out))
    return fail(ctx, LMBR_E_INVALID, "traceback output is NULL");
  const lmbr_config &c = ctx->cfg;
  hipError_t e = lmbr::launch_traceback(c.B, c.K, c.T_max, st->t, c.eos_id, step_opts(ctx, st, ctx->eosx), st->bp, st->tok,
                                        st->qhist, tokens_out, len_out, score_out, step_out, slot_out, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "traceback launch");
  return LMBR_OK;
}

}  // extern "C"

namespace {

// T steps of the decode loop (the model's decoder states -- state_fn, or the
// built-in stand-in -- then the step and the merge) on `stream`.
int32_t decode_loop(lmbr_ctx *ctx, lmbr_beam_state *st, int32_t T, lmbr_state_fn state_fn, void *user,
                    const float *eos_bias, hipStream_t stream) {
  const lmbr_config &c = ctx->cfg;
  for (int32_t i = 0; i < T; ++i) {
    if (state_fn) {
      const int32_t r = state_fn(user, st->t, st, ctx->hidden, stream);
      if (r != 0) return fail(ctx, r, "state_fn returned %d at step %d", r, st->t);
    } else {
      hipError_t e = lmbr::launch_synth_hidden(st->hhash, ctx->hidden, ctx->M, c.H, stream);
      if (e != hipSuccess) return hip_fail(ctx, e, "synth launch");
    }
    int32_t rc = score_step(ctx, st, ctx->hidden, eos_bias ? eos_bias + (size_t)i * c.B : nullptr, stream);
    if (rc == LMBR_OK) rc = merge_step(ctx, st, ws_partials(ctx), ctx->strips, nullptr, nullptr, nullptr, stream);
    if (rc) return rc;
  }
  return LMBR_OK;
}

lmbr_ctx::DecodeKey decode_key(const lmbr_ctx *ctx, const lmbr_beam_state *st, int32_t T, const float *eos_bias) {
  lmbr_ctx::DecodeKey k;
  k.T = T;
  k.t0 = st->t;
  k.st = *st;
  k.st.t = 0;
  k.eos_bias = eos_bias;
  k.W = ctx->W;
  k.bias = ctx->bias;
  k.step_path = ctx->step_path;
  k.length_norm = ctx->length_norm;
  k.finish = ctx->finish;
  k.early_prune = ctx->early_prune;
  k.prune_width = ctx->prune_width;
  k.has_steps = ctx->has_steps;
  k.allowed = ctx->allowed;
  return k;
}

bool same_key(const lmbr_ctx::DecodeKey &a, const lmbr_ctx::DecodeKey &b) {
  return a.T == b.T && a.t0 == b.t0 && a.st.q == b.st.q && a.st.ctx == b.st.ctx && a.st.hhash == b.st.hhash &&
         a.st.len == b.st.len && a.st.ranges == b.st.ranges && a.st.bp == b.st.bp && a.st.tok == b.st.tok &&
         a.st.qhist == b.st.qhist && a.st.sent == b.st.sent && a.eos_bias == b.eos_bias && a.W == b.W &&
         a.bias == b.bias && a.step_path == b.step_path && a.length_norm == b.length_norm &&
         a.finish == b.finish && a.early_prune == b.early_prune && a.prune_width == b.prune_width &&
         a.has_steps == b.has_steps && a.allowed == b.allowed;
}

// The decode loop as a HIP graph: captured on the context's private stream at
// the first call with a given key (the arguments and options it bakes in),
// then replayed on the caller's stream, which saves the per-kernel launch gaps
// of T x 4 dependent launches.  The context keeps the graphs of its last few
// keys (a caller decoding in chunks of a few lengths keeps all of them).
// Falls back to launching the loop directly when the caller's stream is
// itself being captured or a graph cannot be built.
int32_t decode_steps(lmbr_ctx *ctx, lmbr_beam_state *st, int32_t T, const float *eos_bias, hipStream_t stream) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone)
    return decode_loop(ctx, st, T, nullptr, nullptr, eos_bias, stream);
  const lmbr_ctx::DecodeKey key = decode_key(ctx, st, T, eos_bias);
  lmbr_ctx::DecodeGraph *hit = nullptr, *victim = &ctx->graphs[0];
  for (auto &g : ctx->graphs) {
    if (g.exec && same_key(key, g.key)) hit = &g;
    if (!g.exec || (victim->exec && g.last_use < victim->last_use)) victim = &g;
  }
  if (!hit) {
    if (victim->exec) {
      LMBR_HIP(ctx, hipDeviceSynchronize());        // no replay of the replaced graph in flight
      (void)hipGraphExecDestroy(victim->exec);
      victim->exec = nullptr;
    }
    if (!ctx->cap_stream) LMBR_HIP(ctx, hipStreamCreateWithFlags(&ctx->cap_stream, hipStreamNonBlocking));
    const int32_t t0 = st->t;
    if (hipStreamBeginCapture(ctx->cap_stream, hipStreamCaptureModeThreadLocal) != hipSuccess) {
      (void)hipGetLastError();
      return decode_loop(ctx, st, T, nullptr, nullptr, eos_bias, stream);
    }
    const int32_t rc = decode_loop(ctx, st, T, nullptr, nullptr, eos_bias, ctx->cap_stream);
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(ctx->cap_stream, &g);
    hipGraphExec_t x = nullptr;
    const bool built = rc == LMBR_OK && e == hipSuccess && g &&
                       hipGraphInstantiate(&x, g, nullptr, nullptr, 0) == hipSuccess;
    if (g) (void)hipGraphDestroy(g);
    if (!built) {
      (void)hipGetLastError();
      st->t = t0;
      ctx->scored = false;
      if (rc) return rc;
      return decode_loop(ctx, st, T, nullptr, nullptr, eos_bias, stream);
    }
    victim->exec = x;
    victim->key = key;
    hit = victim;
  } else {
    // the host-side effects of the captured steps
    st->t += T;
    ctx->scored = false;
    ctx->strips = ctx->step_path == LMBR_STEP_FUSED ? ctx->sp.fused_strips : ctx->sp.score_strips;
  }
  hit->last_use = ++ctx->graph_clock;
  const hipError_t e = hipGraphLaunch(hit->exec, stream);
  if (e != hipSuccess) return hip_fail(ctx, e, "decode graph launch");
  return LMBR_OK;
}

}  // namespace

extern "C" {

int32_t lmbr_decode(lmbr_ctx *ctx, lmbr_beam_state *st, int32_t T, lmbr_state_fn state_fn, void *user,
                    const float *eos_bias, int32_t *tokens_out, int32_t *len_out, double *score_out,
                    hipStream_t stream) {
  if (!ctx) return LMBR_E_INVALID;
  int32_t rc = check_state(ctx, st);
  if (rc) return rc;
  if (!ctx->W) return fail(ctx, LMBR_E_STATE, "no projection set (lmbr_set_projection)");
  if (T < 0 || st->t + T > ctx->cfg.T_max)
    return fail(ctx, LMBR_E_STATE, "t=%d + T=%d exceeds T_max=%d", st->t, T, ctx->cfg.T_max);
  if (bad_ptr(tokens_out) || bad_ptr(len_out) || bad_ptr(score_out))
    return fail(ctx, LMBR_E_INVALID, "decode output is NULL");
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone)
    return fail(ctx, LMBR_E_STATE, "lmbr_decode synchronises: not for a stream under capture");
  if (T > 0) {
    rc = state_fn ? decode_loop(ctx, st, T, state_fn, user, eos_bias, stream)
                  : decode_steps(ctx, st, T, eos_bias, stream);
    if (rc) return rc;
  }
  if ((rc = lmbr_traceback(ctx, st, ctx->tb_tok, ctx->tb_len, ctx->tb_score, nullptr, nullptr, stream))) return rc;
  const lmbr_config &c = ctx->cfg;
  LMBR_HIP(ctx, hipMemcpyAsync(tokens_out, ctx->tb_tok, sizeof(int32_t) * c.B * (size_t)c.T_max,
                               hipMemcpyDeviceToHost, stream));
  LMBR_HIP(ctx, hipMemcpyAsync(len_out, ctx->tb_len, sizeof(int32_t) * c.B, hipMemcpyDeviceToHost, stream));
  LMBR_HIP(ctx, hipMemcpyAsync(score_out, ctx->tb_score, sizeof(double) * c.B, hipMemcpyDeviceToHost, stream));
  return lmbr_device_status(ctx, nullptr, stream);     // waits for the stream once
}

int32_t lmbr_gather_rows(void *dst, const void *src, const int32_t *rows, int32_t n, size_t row_bytes,
                         hipStream_t stream) {
  g_create_err.clear();
  if (n < 0 || (n > 0 && (!dst || !src || !rows)) || row_bytes % 4 != 0 || row_bytes == 0)
    return fail(nullptr, LMBR_E_INVALID, "lmbr_gather_rows: bad arguments");
  hipError_t e = lmbr::launch_gather_rows(dst, src, rows, n, (int64_t)row_bytes, stream);
  if (e != hipSuccess) return fail(nullptr, LMBR_E_HIP, "gather launch: %s", hipGetErrorString(e));
  return LMBR_OK;
}

}  // extern "C"
