// Target-decoupled decoding with a producer on the same GPU (declared in
// include/as2d.h as as2d_run_decoupled).
//
// The producer is a drafter model in its own context (its own HIP stream):
// each of its steps is one greedy decode step of that model on its own
// request, so it conditions only on its own output and never on the
// target's (Section 4.1, "Target-decoupled drafting").  The token it
// publishes for step i is draft[i], supplied by the caller, so that a
// synthetic draft of known quality can be driven by real drafter compute.
// Tokens are published in batches of eight (Appendix C.1).  The verifier
// decodes from the candidate buffer (as2d_verify_from_buffer) until the
// requested number of target tokens is committed.
//
// concurrent = 1: the producer runs in a thread of its own and never waits
// for the verifier; the verifier never waits for the producer (a K1 step
// when nothing is ready).  concurrent = 0: the serial comparator on one
// thread: before each verification the producer generates whole batches
// until `budget` candidates past the cursor are published (or the draft is
// exhausted), so the two never overlap.
//
// Graphs are captured for both contexts before the producer thread starts,
// so no two threads ever capture at the same time.
//
// Every producer step and verifier call is logged as a closed interval
// (host steady clock, ns from the start of the run); the run ends when
// both sides have stopped (the producer's drain included).

#include <algorithm>
#include <atomic>
#include <chrono>
#include <thread>
#include <vector>

#include "../../include/as2d.h"
#include "internal.h"

namespace {

int64_t now_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now().time_since_epoch())
      .count();
}

struct Log {
  as2d_interval* out;
  int32_t cap;
  std::atomic<int32_t> n{0};
  std::atomic<bool> overflow{false};
  void add(int64_t t0, int64_t s, int64_t e, int32_t kind, int32_t tokens) {
    const int32_t i = n.fetch_add(1);
    if (i >= cap) {
      overflow.store(true);
      return;
    }
    out[i] = as2d_interval{s - t0, e - t0, kind, tokens};
  }
};

// One producer step: a decode step of the drafter, then (every eighth token
// or at the end of the draft) a published batch.
struct Producer {
  as2d_ctx* ctx;
  int32_t req;
  const int32_t* draft;
  int32_t n_draft;
  as2d_cbuf* buf;
  int32_t next = 0;     // draft tokens generated
  int32_t pending = 0;  // generated, not yet published
  int rc = AS2D_OK;
  int step(Log& log, int64_t t0) {
    const int64_t s = now_ns();
    as2d_verify_out o;
    int r = as2d_decode_one(ctx, req, &o);
    if (r == AS2D_OK) {
      ++next;
      ++pending;
      if (pending == 8 || next == n_draft) {
        r = as2d_cbuf_publish(buf, draft + (next - pending), pending, 0, 1, next - pending, now_ns() - t0,
                              __builtin_nanf(""), nullptr);
        pending = 0;
      }
    }
    log.add(t0, s, now_ns(), 0, 1);
    return r;
  }
};

}  // namespace

extern "C" int as2d_run_decoupled(as2d_ctx* target, int32_t treq, as2d_ctx* drafter, int32_t dreq,
                                  const int32_t* draft, int32_t n_draft, int32_t budget, int32_t n_commit,
                                  int32_t concurrent, as2d_cbuf* buf, as2d_read_cursor* cur, int32_t* committed,
                                  as2d_interval* log, int32_t log_cap, int32_t* n_log, int64_t* total_ns,
                                  int32_t* producer_rc) {
  if (!target || !drafter || !buf || !cur || !committed || !log || !n_log || !total_ns || n_commit < 1 ||
      budget < 0 || n_draft < 0 || (n_draft > 0 && !draft) || log_cap < 1)
    return AS2D_EINVAL;
  int64_t pub = 0;
  as2d_cbuf_snapshot(buf, &pub);
  if (pub != 0 || cur->cursor != 0) return AS2D_EINVAL;   // a fresh buffer and cursor
  // every graph either thread will launch is captured here, one context
  // at a time, before the producer thread starts: the target's passes of
  // 1..budget + 1 rows and the drafter's one-row decode step
  int prc = as2d_prepare_graphs(target, budget + 1);
  if (prc == AS2D_OK) prc = as2d_prepare_graphs(drafter, 1);
  if (prc != AS2D_OK) return prc;
  Log lg{log, log_cap};
  Producer prod{drafter, dreq, draft, n_draft, buf};
  std::atomic<bool> stop{false};
  int rc = AS2D_OK;
  int32_t got = 0;
  const int64_t t0 = now_ns();

  auto verify = [&]() {
    const int64_t s = now_ns();
    const int64_t c0 = cur->cursor;
    as2d_verify_out o;
    int32_t k = 0;
    int r = as2d_verify_from_buffer(target, treq, buf, cur, budget, n_commit - got, &o, &k);
    if (r != AS2D_OK) return r;
    if (o.accepted_len) r = as2d_cbuf_read(buf, c0, o.accepted_len, committed + got);
    got += o.accepted_len;
    committed[got++] = o.correction_token;
    lg.add(t0, s, now_ns(), 1, o.accepted_len + 1);
    return r;
  };

  if (concurrent) {
    std::thread th([&] {
      while (!stop.load(std::memory_order_relaxed) && prod.next < n_draft) {
        const int r = prod.step(lg, t0);
        if (r != AS2D_OK) {
          prod.rc = r;
          break;
        }
      }
    });
    while (got < n_commit && rc == AS2D_OK) rc = verify();
    stop.store(true);
    th.join();
  } else {
    while (got < n_commit && rc == AS2D_OK) {
      int64_t n = 0;
      as2d_cbuf_snapshot(buf, &n);
      while (prod.rc == AS2D_OK && prod.next < n_draft && (n < cur->cursor + budget || prod.pending)) {
        prod.rc = prod.step(lg, t0);
        as2d_cbuf_snapshot(buf, &n);
      }
      rc = verify();
    }
  }
  *total_ns = now_ns() - t0;
  *n_log = std::min(lg.n.load(), log_cap);
  if (producer_rc) *producer_rc = prod.rc;
  if (rc == AS2D_OK && lg.overflow.load()) rc = AS2D_ECAPACITY;
  return rc;
}
