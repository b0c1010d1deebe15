// Host construction of one sentence's posterior table.
//
// Section 2 of the paper arranges L as a matrix with one row per n-gram
// history and one column per vocabulary word; only the posterior part of a row
// is sparse (theta0 makes it dense).  The table built here is that sparse part:
// every (n-1)-word history of the sentence's evidence space maps, through an
// open-addressed hash, to the list of its successor words and their posteriors
// (Eq. 2's P_LMBR).  The sparse layout applies theta0 and the theta_n weights
// on the GPU on the fly (the library keeps only the history-free part of L as
// one dense row per sentence); lmbr_table_dense builds the paper's own dense
// arrangement, one row per history, for small evidence spaces.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "lmbr.h"
#include "tables.h"

namespace lmbr {

uint64_t pack_context(const int32_t *words, int n_words) {
  uint64_t key = 0;
  for (int i = 0; i < n_words; ++i) key = (key << kWordBits) | (uint64_t)(words[i] + 1);
  return key;
}

}  // namespace lmbr

namespace {

struct Rec {
  uint64_t key;  // packed history (empty history = 0)
  int32_t tok;   // last word of the n-gram
  float post;
};

void set_err(char *err, size_t err_len, const char *msg) {
  if (err && err_len) {
    std::strncpy(err, msg, err_len - 1);
    err[err_len - 1] = '\0';
  }
}

}  // namespace

extern "C" int32_t lmbr_table_build(int32_t V, int64_t n, const int32_t *order,
                                    const int32_t *tokens, const float *post, float load_factor,
                                    lmbr_table_image *out, char *err, size_t err_len) {
  char msg[256];
  if (!out) {
    set_err(err, err_len, "lmbr_table_build: out is NULL");
    return LMBR_E_INVALID;
  }
  std::memset(out, 0, sizeof(*out));
  if (V < 2 || V > LMBR_MAX_V) {
    std::snprintf(msg, sizeof msg, "lmbr_table_build: V=%d outside [2, %d]", V, LMBR_MAX_V);
    set_err(err, err_len, msg);
    return LMBR_E_INVALID;
  }
  if (n < 0 || n > (int64_t)INT32_MAX) {
    set_err(err, err_len, "lmbr_table_build: n outside [0, 2^31)");
    return LMBR_E_INVALID;
  }
  if (n > 0 && (!order || !tokens || !post)) {
    set_err(err, err_len, "lmbr_table_build: NULL array with n > 0");
    return LMBR_E_INVALID;
  }
  if (load_factor == 0.f) load_factor = 0.5f;
  if (!(load_factor > 0.f && load_factor <= 0.9f)) {
    set_err(err, err_len, "lmbr_table_build: load_factor outside (0, 0.9]");
    return LMBR_E_INVALID;
  }

  std::vector<Rec> recs((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    const int o = order[i];
    if (o < 1 || o > LMBR_MAX_ORDER) {
      std::snprintf(msg, sizeof msg, "lmbr_table_build: n-gram %lld has order %d outside 1..4",
                    (long long)i, o);
      set_err(err, err_len, msg);
      return LMBR_E_INVALID;
    }
    const int32_t *w = tokens + 4 * i;
    for (int j = 0; j < o; ++j) {
      if (w[j] < 0 || w[j] >= V) {
        std::snprintf(msg, sizeof msg, "lmbr_table_build: n-gram %lld has word %d outside [0, %d)",
                      (long long)i, w[j], V);
        set_err(err, err_len, msg);
        return LMBR_E_INVALID;
      }
    }
    const float p = post[i];
    if (!(p > 0.f && p <= 1.f)) {
      std::snprintf(msg, sizeof msg, "lmbr_table_build: n-gram %lld has posterior %g outside (0, 1]",
                    (long long)i, (double)p);
      set_err(err, err_len, msg);
      return LMBR_E_INVALID;
    }
    recs[(size_t)i] = Rec{lmbr::pack_context(w, o - 1), w[o - 1], p};
  }
  std::sort(recs.begin(), recs.end(), [](const Rec &a, const Rec &b) {
    return a.key != b.key ? a.key < b.key : a.tok < b.tok;
  });

  int64_t n_ctx = 0;  // histories of orders 2..4 (the empty history is kept apart)
  for (size_t i = 0; i < recs.size(); ++i) {
    if (i > 0 && recs[i].key == recs[i - 1].key && recs[i].tok == recs[i - 1].tok) {
      set_err(err, err_len, "lmbr_table_build: duplicate n-gram");
      return LMBR_E_INVALID;
    }
    if ((i == 0 || recs[i].key != recs[i - 1].key) && recs[i].key != 0) ++n_ctx;
  }

  int64_t cap = 2;
  const double need = std::ceil((double)n_ctx / (double)load_factor);
  while ((double)cap < need || cap <= n_ctx) cap <<= 1;

  out->n_slots = cap;
  out->n_entries = (int64_t)recs.size();
  out->slot_key = (uint64_t *)std::malloc(sizeof(uint64_t) * (size_t)cap);
  out->slot_off = (uint32_t *)std::calloc((size_t)cap, sizeof(uint32_t));
  out->slot_cnt = (uint32_t *)std::calloc((size_t)cap, sizeof(uint32_t));
  out->entry_tok = (int32_t *)std::malloc(sizeof(int32_t) * std::max<size_t>(1, recs.size()));
  out->entry_post = (float *)std::malloc(sizeof(float) * std::max<size_t>(1, recs.size()));
  if (!out->slot_key || !out->slot_off || !out->slot_cnt || !out->entry_tok || !out->entry_post) {
    lmbr_table_free(out);
    set_err(err, err_len, "lmbr_table_build: host out of memory");
    return LMBR_E_CAPACITY;
  }
  for (int64_t i = 0; i < cap; ++i) out->slot_key[i] = lmbr::kEmptyKey;

  const uint64_t mask = (uint64_t)cap - 1;
  size_t i = 0;
  while (i < recs.size()) {
    size_t j = i;
    while (j < recs.size() && recs[j].key == recs[i].key) {
      out->entry_tok[j] = recs[j].tok;
      out->entry_post[j] = recs[j].post;
      ++j;
    }
    if (recs[i].key == 0) {
      out->uni_off = (uint32_t)i;
      out->uni_cnt = (uint32_t)(j - i);
    } else {
      uint64_t h = lmbr::splitmix64(recs[i].key) & mask;
      while (out->slot_key[h] != lmbr::kEmptyKey) h = (h + 1) & mask;
      out->slot_key[h] = recs[i].key;
      out->slot_off[h] = (uint32_t)i;
      out->slot_cnt[h] = (uint32_t)(j - i);
    }
    i = j;
  }
  set_err(err, err_len, "");
  return LMBR_OK;
}

extern "C" void lmbr_table_free(lmbr_table_image *img) {
  if (!img) return;
  std::free(img->slot_key);
  std::free(img->slot_off);
  std::free(img->slot_cnt);
  std::free(img->entry_tok);
  std::free(img->entry_post);
  std::memset(img, 0, sizeof(*img));
}

namespace {

// The slot of a packed history in the image's hash, or -1 (host mirror of the
// device probe: slot = SplitMix64(key) & (capacity - 1), linear probing).
int64_t find_slot(const lmbr_table_image *img, uint64_t key) {
  const uint64_t mask = (uint64_t)img->n_slots - 1;
  uint64_t h = lmbr::splitmix64(key) & mask;
  for (int64_t step = 0; step < img->n_slots; ++step) {
    if (img->slot_key[h] == key) return (int64_t)h;
    if (img->slot_key[h] == lmbr::kEmptyKey) return -1;
    h = (h + 1) & mask;
  }
  return -1;
}

}  // namespace

extern "C" int64_t lmbr_table_history_count(const lmbr_table_image *img) {
  if (!img || !img->slot_key) return 0;
  int64_t n = 0;
  for (int64_t i = 0; i < img->n_slots; ++i) n += img->slot_key[i] != lmbr::kEmptyKey;
  return n;
}

extern "C" int32_t lmbr_table_dense(const lmbr_table_image *img, int32_t V, int64_t ld, float lambda,
                                    const float *theta, float *rows_out, uint32_t *slot_row_out) {
  if (!img || !img->slot_key || !theta || !rows_out || !slot_row_out || V < 2 || ld < V)
    return LMBR_E_INVALID;
  // rows: 0 = the empty history, then the occupied slots in slot order
  int64_t nrows = 1;
  for (int64_t i = 0; i < img->n_slots; ++i)
    slot_row_out[i] = img->slot_key[i] != lmbr::kEmptyKey ? (uint32_t)nrows++ : UINT32_MAX;
  std::vector<double> acc((size_t)V, 0.0);
  std::vector<char> seen((size_t)V, 0);
  std::vector<int32_t> touched;
  auto emit = [&](int64_t r, uint64_t key) {
    // the history's words: its 21-bit fields, newest lowest; a history of l
    // words gets the orders n = 1 .. l + 1, each from the successors of its
    // last n - 1 words (Eq. 2), all weighted by lambda (theta0 is added on
    // the device after the upload, as the paper does)
    int l = 0;
    while (l < 3 && ((key >> (lmbr::kWordBits * l)) & ((1ull << lmbr::kWordBits) - 1)) != 0) ++l;
    for (int n = 1; n <= l + 1; ++n) {
      uint32_t off = 0, cnt = 0;
      if (n == 1) {
        off = img->uni_off;
        cnt = img->uni_cnt;
      } else {
        const uint64_t sub = key & ((1ull << (lmbr::kWordBits * (n - 1))) - 1);
        const int64_t h = find_slot(img, sub);
        if (h < 0) continue;
        off = img->slot_off[h];
        cnt = img->slot_cnt[h];
      }
      for (uint32_t k = 0; k < cnt; ++k) {
        const int32_t y = img->entry_tok[off + k];
        if (!seen[(size_t)y]) {
          seen[(size_t)y] = 1;
          touched.push_back(y);
        }
        acc[(size_t)y] += (double)theta[n] * (double)img->entry_post[off + k];
      }
    }
    float *row = rows_out + r * ld;
    std::memset(row, 0, sizeof(float) * (size_t)ld);
    for (int32_t y : touched) {
      row[y] = (float)((double)lambda * acc[(size_t)y]);
      acc[(size_t)y] = 0.0;
      seen[(size_t)y] = 0;
    }
    touched.clear();
  };
  emit(0, 0);
  for (int64_t i = 0; i < img->n_slots; ++i)
    if (img->slot_key[i] != lmbr::kEmptyKey) emit(slot_row_out[i], img->slot_key[i]);
  return LMBR_OK;
}

extern "C" int32_t lmbr_plan_batches(int64_t n, const int32_t *lengths, int32_t B, int32_t sorted,
                                     int64_t *order_out, int32_t *batch_steps_out) {
  if (n < 0 || B < 1 || (n > 0 && (!lengths || !order_out || !batch_steps_out))) return LMBR_E_INVALID;
  for (int64_t i = 0; i < n; ++i)
    if (lengths[i] < 1) return LMBR_E_INVALID;
  std::vector<int64_t> idx((size_t)n);
  for (int64_t i = 0; i < n; ++i) idx[(size_t)i] = i;
  if (sorted)
    std::stable_sort(idx.begin(), idx.end(), [&](int64_t a, int64_t b) { return lengths[a] > lengths[b]; });
  for (int64_t i = 0; i < n; ++i) order_out[i] = idx[(size_t)i];
  for (int64_t b0 = 0; b0 < n; b0 += B) {
    int32_t m = 0;
    for (int64_t i = b0; i < std::min<int64_t>(n, b0 + B); ++i) m = std::max(m, lengths[idx[(size_t)i]]);
    batch_steps_out[b0 / B] = m;
  }
  return LMBR_OK;
}
