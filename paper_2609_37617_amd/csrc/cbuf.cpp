// Candidate buffer, read cursor and candidate alignment (host side of the
// decoding loop; declared in include/as2d.h).
//
// Ordered publication (Section 4.1, "Ordered publication and buffering";
// Appendix C.1): one producer appends immutable batches of up to eight
// tokens with their provenance; readers see a prefix of them (a snapshot)
// and never block the producer.  Tokens and records live in arrays sized at
// creation; a batch is written first and then made visible by one release
// store of the published length, so a reader that loads the length with
// acquire ordering reads only complete batches.
//
// The read cursor and its realignment (Section 4.2, "Candidate alignment";
// Appendix C.3; Figure 4(c)) are a pure function of the snapshot and the
// verification outcome; the rule is stated at as2d_cursor_update in the
// header.

#include <atomic>
#include <cstring>
#include <memory>
#include <new>

#include "../../include/as2d.h"

struct as2d_cbuf {
  int64_t capacity = 0;
  std::unique_ptr<int32_t[]> tokens;
  std::unique_ptr<as2d_cbuf_record[]> records;
  std::atomic<int64_t> published{0};
  std::atomic<int64_t> n_records{0};
};

namespace {
constexpr int32_t kBatch = 8;
constexpr int32_t kMaxRadius = 64;
}  // namespace

extern "C" {

int as2d_cbuf_create(int64_t capacity, as2d_cbuf** out) {
  if (!out || capacity < 1 || capacity > (int64_t(1) << 31)) return AS2D_EINVAL;
  as2d_cbuf* b = new (std::nothrow) as2d_cbuf;
  if (!b) return AS2D_ENOMEM;
  b->tokens.reset(new (std::nothrow) int32_t[capacity]);
  b->records.reset(new (std::nothrow) as2d_cbuf_record[capacity]);
  if (!b->tokens || !b->records) {
    delete b;
    return AS2D_ENOMEM;
  }
  b->capacity = capacity;
  *out = b;
  return AS2D_OK;
}

int as2d_cbuf_free(as2d_cbuf* b) {
  delete b;
  return AS2D_OK;
}

int as2d_cbuf_publish(as2d_cbuf* b, const int32_t* tokens, int32_t n, int32_t source_id, int32_t producer_id,
                      int64_t offset, int64_t publish_ns, float confidence, int64_t* published) {
  if (!b || !tokens || n < 1 || n > kBatch) return AS2D_EINVAL;
  const int64_t first = b->published.load(std::memory_order_relaxed);   // only the producer writes it
  const int64_t r = b->n_records.load(std::memory_order_relaxed);
  if (first + n > b->capacity) return AS2D_ECAPACITY;
  std::memcpy(b->tokens.get() + first, tokens, sizeof(int32_t) * n);
  as2d_cbuf_record& rec = b->records[r];
  rec.first = first;
  rec.count = n;
  rec.source_id = source_id;
  rec.producer_id = producer_id;
  rec.pad = 0;
  rec.offset = offset;
  rec.publish_ns = publish_ns;
  rec.confidence = confidence;
  rec.pad2 = 0;
  b->n_records.store(r + 1, std::memory_order_release);
  b->published.store(first + n, std::memory_order_release);
  if (published) *published = first + n;
  return AS2D_OK;
}

int as2d_cbuf_snapshot(const as2d_cbuf* b, int64_t* n) {
  if (!b || !n) return AS2D_EINVAL;
  *n = b->published.load(std::memory_order_acquire);
  return AS2D_OK;
}

int as2d_cbuf_read(const as2d_cbuf* b, int64_t start, int32_t n, int32_t* out) {
  if (!b || (n > 0 && !out) || start < 0 || n < 0) return AS2D_EINVAL;
  if (n > 0 && start + n > b->published.load(std::memory_order_acquire)) return AS2D_EINVAL;
  if (n) std::memcpy(out, b->tokens.get() + start, sizeof(int32_t) * n);
  return AS2D_OK;
}

int as2d_cbuf_n_records(const as2d_cbuf* b, int64_t* n) {
  if (!b || !n) return AS2D_EINVAL;
  *n = b->n_records.load(std::memory_order_acquire);
  return AS2D_OK;
}

int as2d_cbuf_get_record(const as2d_cbuf* b, int64_t i, as2d_cbuf_record* out) {
  if (!b || !out || i < 0 || i >= b->n_records.load(std::memory_order_acquire)) return AS2D_EINVAL;
  *out = b->records[i];
  return AS2D_OK;
}

int as2d_cursor_init(as2d_read_cursor* c, int32_t radius) {
  if (!c || radius < 0 || radius > kMaxRadius) return AS2D_EINVAL;
  c->cursor = 0;
  c->floor = 0;
  c->radius = radius;
  c->pad = 0;
  return AS2D_OK;
}

int as2d_cursor_propose(const as2d_cbuf* b, const as2d_read_cursor* c, int64_t snapshot, int32_t k_max,
                        int32_t* cands, int32_t* k) {
  if (!b || !c || !k || k_max < 0 || (k_max > 0 && !cands)) return AS2D_EINVAL;
  if (snapshot < 0 || snapshot > b->published.load(std::memory_order_acquire)) return AS2D_EINVAL;
  int64_t n = snapshot - c->cursor;
  if (n < 0) n = 0;
  if (n > k_max) n = k_max;
  if (n) std::memcpy(cands, b->tokens.get() + c->cursor, sizeof(int32_t) * n);
  *k = (int32_t)n;
  return AS2D_OK;
}

int as2d_cursor_update(const as2d_cbuf* b, as2d_read_cursor* c, int64_t snapshot, int32_t k, int32_t accepted,
                       int32_t token) {
  if (!b || !c || k < 0 || accepted < 0 || accepted > k) return AS2D_EINVAL;
  if (snapshot < 0 || snapshot > b->published.load(std::memory_order_acquire)) return AS2D_EINVAL;
  const int32_t* t = b->tokens.get();
  const int64_t m = c->cursor + accepted;   // the position the committed token stands for
  if (accepted > 0) c->floor = m;
  if (m < snapshot && t[m] == token) {
    c->cursor = c->floor = m + 1;
    return AS2D_OK;
  }
  for (int32_t d = 1; d <= c->radius; ++d) {
    const int64_t fwd = m + d, bwd = m - d;
    if (fwd < snapshot && t[fwd] == token) {
      c->cursor = c->floor = fwd + 1;
      return AS2D_OK;
    }
    if (bwd >= c->floor && bwd < snapshot && t[bwd] == token) {
      c->cursor = c->floor = bwd + 1;
      return AS2D_OK;
    }
  }
  c->cursor = m + 1;   // substitution: position m stays eligible (floor unchanged)
  return AS2D_OK;
}

int as2d_verify_from_buffer(as2d_ctx* ctx, int32_t req, const as2d_cbuf* b, as2d_read_cursor* c, int32_t budget,
                            int32_t max_commit, as2d_verify_out* out, int32_t* k_used) {
  if (!ctx || !b || !c || !out || budget < 0 || max_commit < 1) return AS2D_EINVAL;
  int32_t cands[AS2D_MAX_BUDGET];
  int32_t k_max = budget < max_commit - 1 ? budget : max_commit - 1;
  if (k_max > AS2D_MAX_BUDGET) k_max = AS2D_MAX_BUDGET;
  int64_t n = 0;
  int32_t k = 0;
  int rc = as2d_cbuf_snapshot(b, &n);
  if (rc == AS2D_OK) rc = as2d_cursor_propose(b, c, n, k_max, cands, &k);
  if (rc != AS2D_OK) return rc;
  as2d_verify_out r;
  rc = as2d_verify(ctx, req, k ? cands : nullptr, k, &r);
  if (rc != AS2D_OK) return rc;
  rc = as2d_cbuf_snapshot(b, &n);
  if (rc == AS2D_OK) rc = as2d_cursor_update(b, c, n, k, r.accepted_len, r.correction_token);
  if (rc != AS2D_OK) return rc;
  *out = r;
  if (k_used) *k_used = k;
  return AS2D_OK;
}

}  // extern "C"
