/*
 * as2d.h - C ABI of the MI355X (gfx950) target verification library.
 *
 * The library runs the target side of AS2D's decoding loop (arXiv
 * 2609.37617): a decoder-only target model, prefilled with audio
 * embeddings and instruction tokens, verifies a known root token plus k
 * drafted candidates in one forward pass and commits the longest prefix of
 * candidates equal to its own greedy tokens, followed by its correction
 * (Section 4.2 "Target verification"; Appendix C.2 "Verification and state
 * repair").  Rejected cache entries are dropped by shortening the logical
 * KV length; nothing is copied.
 *
 * Conventions for every call:
 *   - Return value: AS2D_OK (0) or a negative AS2D_E* code.  Outputs are
 *     written only on success; on failure as2d_last_error(ctx) holds a
 *     message (for a failed as2d_load_weights, which leaves no context,
 *     as2d_last_error(NULL) on the same thread).
 *   - Host pointers are owned by the caller and only read (or written, for
 *     outputs) during the call; the library copies what it keeps.
 *   - All device memory (packed weights, KV cache slots, scratch) is owned
 *     by the library and released by as2d_free().
 *   - Number formats: weights are stored in cfg->dtype; the residual
 *     stream, softmax and accumulators are float32, and bf16 models
 *     multiply activations into the weights as bf16 (hi, lo) pairs, i.e.
 *     to about 17 significant bits; their KV cache holds the keys and
 *     values as such pairs too (4 bytes per element, as float32).
 *   - A context is used by one host thread at a time.
 *   - Token ids are int32 in [0, vocab).
 *
 * Model: pre-RMSNorm decoder layers with grouped-query attention (query
 * head h reads KV head floor(h * n_kv / n_q)), rotary position embedding
 * (rotate-half pairs (i, i + d/2), angle pos * theta^(-2i/d)), optional QKV
 * bias, SwiGLU MLP, final RMSNorm and an untied LM head.  The greedy token
 * is the arg-max logit, ties to the lowest token id (the deterministic
 * tie-break of Appendix C.4, Eq. reference-transition).
 */
#ifndef AS2D_H
#define AS2D_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  AS2D_OK = 0,
  AS2D_EINVAL = -1,    /* bad argument: k, token id, request id, rollback length, null pointer */
  AS2D_ECAPACITY = -2, /* the request's KV slot cannot hold the new rows */
  AS2D_ESTATE = -3,    /* verify/decode on a request that has not been prefilled */
  AS2D_EHIP = -4,      /* HIP runtime error */
  AS2D_ENUMERIC = -5,  /* non-finite logits: no token can be chosen */
  AS2D_ENOMEM = -6     /* device or pinned host allocation failed */
};

enum { AS2D_F32 = 0, AS2D_BF16 = 1 };

typedef struct as2d_ctx as2d_ctx;

typedef struct {
  int32_t n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab;
  float rope_theta, rms_eps;
  int32_t dtype;    /* AS2D_F32 or AS2D_BF16: weights, GEMM operands and KV cache */
  int32_t qkv_bias; /* 0 or 1 */
  int32_t max_requests, max_kv_len, max_k; /* KV slots, positions per slot, candidates per call */
} as2d_config;

typedef struct {
  int32_t accepted_len;     /* a in [0, k]: candidates committed */
  int32_t correction_token; /* target's greedy token after root + a candidates; the next root */
  int32_t kv_len;           /* positions now in the KV cache: previous kv_len + a + 1 */
  int32_t committed;        /* tokens committed since prefill (first root excluded) */
} as2d_verify_out;

/*
 * Load a model and create a context.
 *
 * host_tensors: n_tensors pointers in this canonical order
 *   embed [vocab][hidden]
 *   per layer l = 0..n_layers-1:
 *     attn_norm [hidden], wq [n_q*d][hidden], wk [n_kv*d][hidden], wv [n_kv*d][hidden],
 *     (qkv_bias only) bq [n_q*d], bk [n_kv*d], bv [n_kv*d],
 *     wo [hidden][n_q*d], mlp_norm [hidden],
 *     w_gate [ffn][hidden], w_up [ffn][hidden], w_down [hidden][ffn]
 *   final_norm [hidden], lm_head [vocab][hidden]
 * Matrices and the embedding are row-major in cfg->dtype (bf16 as uint16
 * bit patterns); norm gains and biases are float32.
 * Shape requirements: head_dim 64 or 128, n_q divisible by n_kv, hidden a
 * multiple of 128, ffn a multiple of 64, vocab a multiple of 128,
 * max_k <= 31, max_kv_len <= 32768, hidden <= 8192.
 * hip_stream: the hipStream_t all work is ordered on (NULL: the library
 * creates its own).  The weights are repacked on the device into the tile
 * order the GEMM kernels stream.
 */
int as2d_load_weights(const as2d_config* cfg, const void* const* host_tensors, int32_t n_tensors,
                      void* hip_stream, as2d_ctx** out);

/*
 * Prefill request slot `req` (Appendix A.1: the prepared audio KV and the
 * instruction give the initial decoding state; Appendix C.2).
 * audio_emb: [n_audio][hidden] in cfg->dtype, used directly as hidden
 * states at positions 0..n_audio-1; instr_tokens: n_instr token ids at the
 * following positions.  n_audio + n_instr >= 1 and <= max_kv_len.
 * On success *first_token is the greedy token after the prefix (the first
 * root, not yet in the cache) and *kv_len = n_audio + n_instr.
 * Re-prefilling a slot discards its previous state.
 */
int as2d_prefill_kv(as2d_ctx* ctx, int32_t req, const void* audio_emb, int32_t n_audio,
                    const int32_t* instr_tokens, int32_t n_instr, int32_t* first_token,
                    int32_t* kv_len);

/*
 * One verification call (Section 4.2; Appendix C.2): the pending root and
 * cands[0..k) are processed at positions kv_len..kv_len+k in one forward
 * pass; accepted_len is the length of the longest candidate prefix equal
 * to the target's greedy tokens and correction_token the greedy token that
 * follows it (a bonus token when all k match).  The root and the accepted
 * candidates stay in the cache; the correction becomes the pending root.
 * 0 <= k <= max_k; kv_len + k + 1 <= max_kv_len (else AS2D_ECAPACITY).
 */
int as2d_verify(as2d_ctx* ctx, int32_t req, const int32_t* cands, int32_t k, as2d_verify_out* out);

/* Target-only (K1) step: as2d_verify with k = 0 (Appendix C.2). */
int as2d_decode_one(as2d_ctx* ctx, int32_t req, as2d_verify_out* out);

/*
 * Verification calls of n distinct requests in one fused forward pass.
 * reqs[i], ks[i] as in as2d_verify; cands_flat holds the requests'
 * candidates back to back (sum of ks entries).  Each request's rows attend
 * only to its own cache slot.  outs[i] receives request i's result.
 * sum(ks[i] + 1) <= 144.
 * Non-finite logits are a per-request outcome: a request with a
 * non-finite logit in any of its rows keeps its state and gets
 * accepted_len = correction_token = -1, the other requests are committed
 * as usual, their outs written, and the call returns AS2D_ENUMERIC
 * (as2d_verify and as2d_decode_one, one request each, then write
 * *out the same way).
 */
int as2d_verify_batch(as2d_ctx* ctx, int32_t n, const int32_t* reqs, const int32_t* cands_flat,
                      const int32_t* ks, as2d_verify_out* outs);

/*
 * Verification for callers that cannot allocate device memory (code under
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * as2d_verify for one request, with every buffer the pass works in
 * (activations, split-K and attention partials, counters, row descriptors)
 * taken from the library's static scratch array (32 MiB per GPU, held until
 * the process ends) instead of the context's own.  The weights, the KV
 * cache, the pinned result buffers and, with keep_logits, the logits stay
 * in the context.  The call allocates nothing and launches its kernels one
 * by one on the context's stream (no graph); results are bit-identical to
 * as2d_verify.  AS2D_ECAPACITY when the pass needs more than the array
 * holds: the need grows with the model's widths and the request's KV length
 * (about 10 MiB for the 7B shape at 1,040 positions); the message gives the
 * bytes.  Every call on one GPU shares the array: calls that overlap on one
 * GPU (from several contexts or threads) race.
 */
int as2d_verify_static(as2d_ctx* ctx, int32_t req, const int32_t* cands, int32_t k, as2d_verify_out* out);

/* ---- test and inspection hooks (not on the timed path) ---------------- */

/* When on, later calls also write the float32 logits of every processed
 * row (off by default). */
int as2d_set_keep_logits(as2d_ctx* ctx, int32_t on);

/* Logits of the rows of `req`'s last verify/decode call (needs
 * keep_logits): host[max_rows][vocab]; *n_rows receives the row count
 * (k + 1).  After a prefill, the logits of the last prefix row. */
int as2d_get_logits(as2d_ctx* ctx, int32_t req, float* host, int32_t max_rows, int32_t* n_rows);

/* Greedy token of every row of `req`'s last call: host[max_rows]. */
int as2d_get_row_tokens(as2d_ctx* ctx, int32_t req, int32_t* host, int32_t max_rows, int32_t* n_rows);

/* Top-2 logit margin of every row of `req`'s last call: host[max_rows]
 * receives the largest logit minus the second-largest (0 when two token
 * ids tie for the maximum), computed on the device beside the arg-max, so
 * a caller can flag near-tied decisions (Appendix F.6 records near-tied
 * top-1 differences across backends) without fetching logits. */
int as2d_get_row_margins(as2d_ctx* ctx, int32_t req, float* host, int32_t max_rows, int32_t* n_rows);

/* How verification passes run; results are bit-identical in every mode.
 *   AS2D_EXEC_EAGER:      one kernel launch per operation (no graph);
 *   AS2D_EXEC_GRAPH:      (default) the same launches captured once per
 *                         (rows, requests, keep_logits) into a HIP graph;
 *   AS2D_EXEC_PERSISTENT: one persistent kernel per pass of up to 32 rows,
 *                         captured into a graph; larger passes use
 *                         AS2D_EXEC_GRAPH.
 * as2d_get_exec_info reports the mode and the persistent kernel's grid
 * (0 when the device, or the compute-unit budget, cannot hold it;
 * verification passes then run as AS2D_EXEC_GRAPH). */
enum { AS2D_EXEC_EAGER = 0, AS2D_EXEC_GRAPH = 1, AS2D_EXEC_PERSISTENT = 2 };
int as2d_set_exec_mode(as2d_ctx* ctx, int32_t mode);
int as2d_get_exec_info(as2d_ctx* ctx, int32_t* mode, int32_t* persistent_grid);

/* Timeline of the persistent step kernel (inspection only): when on, every
 * later persistent pass records, per workgroup and phase, three
 * wall-clock stamps (phase entered, inputs ready, phase left; 0 = not
 * reached).  as2d_step_trace_read copies the last pass's stamps,
 * [grid][n_phase][3] int64, into host (max entries) and reports grid and
 * n_phase.  Phases: 0 embedding; per layer l, 1 + 6 l + {0 QKV,
 * 1 attention chunks, 2 attention merge, 3 O, 4 gate/up, 5 down}; then the
 * LM head and the verification. */
int as2d_set_step_trace(as2d_ctx* ctx, int32_t on);
int as2d_step_trace_read(as2d_ctx* ctx, int64_t* host, int64_t max, int32_t* grid, int32_t* n_phase);

/* Return `req` to an earlier committed state: prefix length <= kv_len <=
 * current kv_len; root becomes the pending root.  Cache rows past kv_len
 * are ignored and overwritten by later calls. */
int as2d_rollback(as2d_ctx* ctx, int32_t req, int32_t kv_len, int32_t root);

/* Current state of `req`: kv_len, pending root and committed count. */
int as2d_get_state(as2d_ctx* ctx, int32_t req, int32_t* kv_len, int32_t* root, int32_t* committed);

/* Copy positions 0..n_tok-1 of one layer's cache: host_k, host_v
 * [n_kv][n_tok][head_dim] float32 (K after rotation).  A bf16 model's
 * cache holds each value as a bf16 pair (hi, lo) with hi + lo equal to the
 * float32 value to about 2^-17 relative (the operands the attention
 * multiplies); that sum is returned.  Float32 models keep float32. */
int as2d_read_kv(as2d_ctx* ctx, int32_t req, int32_t layer, void* host_k, void* host_v, int32_t n_tok);

/* Rebind the context to another stream (hip_stream = NULL: a stream of its
 * own).  Waits for the old stream and drops cached graphs.  A stream
 * confined to part of the device by a CU mask is refused (AS2D_EINVAL);
 * as2d_load_weights refuses one the same way.  Results do not depend on
 * the stream. */
int as2d_set_stream(as2d_ctx* ctx, void* hip_stream);
/* Size the balanced GEMM grids (and the persistent kernel's and the
 * verification attention's) for `cus` compute units (1 .. the device's;
 * 0 restores all of them): each such GEMM then runs cus workgroups of one
 * CU each, and the attention at most cus (two per CU for long caches),
 * leaving the other CUs to work on other streams (a drafter beside the
 * target); prefill kernels still size their grids by the rows.  A GEMM with more
 * than 24 (tile pair, k-split) units per workgroup at that grid keeps the
 * grid that gives it 24; if one does, the persistent kernel (one
 * workgroup per budgeted CU) is not used and as2d_get_exec_info reports
 * grid 0.  Split counts, and so every result, are unchanged.  Waits for
 * the stream and drops cached graphs and per-pass argument arrays. */
int as2d_set_cu_budget(as2d_ctx* ctx, int32_t cus);
/* Mark a slot free (its state is discarded). */
int as2d_release_request(as2d_ctx* ctx, int32_t req);

/*
 * Per-kernel timing with HIP events on the library's stream.  When on,
 * each launch of the step is bracketed by events and its duration is
 * accumulated per kernel kind; this serialises nothing but adds event
 * records between launches.  as2d_timing_read fills up to max entries of
 * names (each up to 31 chars + NUL, 32 bytes per entry), total
 * milliseconds and launch counts, and returns the number of kinds.
 */
int as2d_set_timing(as2d_ctx* ctx, int32_t on);
int as2d_timing_read(as2d_ctx* ctx, char* names, double* total_ms, int64_t* counts, int32_t max);
int as2d_timing_reset(as2d_ctx* ctx);

/* Average duration of one GEMM kernel of kind `which` (0 QKV, 1 O,
 * 2 gate/up, 3 down, 4 LM head) for `rows` rows, from `reps` back-to-back
 * launches on the library's stream between two HIP events; the layer
 * matrices are cycled so the weights stream from HBM.  Measurement only:
 * it overwrites activation buffers and the cache rows 0..rows-1 of slot 0. */
int as2d_time_gemm(as2d_ctx* ctx, int32_t which, int32_t rows, int32_t reps, double* avg_us);

/* Achievable read bandwidth of the device, the ceiling for weight-streaming
 * kernels: a plain kernel streams `bytes` (rounded down to a multiple of
 * 64 MiB, at least 64 MiB) of a scratch buffer with 16-byte non-temporal
 * loads, one workgroup per compute unit and 32 KiB in flight per unit;
 * `reps` back-to-back launches between two HIP events on the library's
 * stream.  Writes GB/s (1e9 bytes per second) to *gbps.  Allocates and
 * frees the scratch buffer inside the call; EINVAL for bytes < 64 MiB or
 * reps < 1, ENOMEM if the buffer does not fit. */
int as2d_stream_bandwidth(as2d_ctx* ctx, int64_t bytes, int32_t reps, double* gbps);

/*
 * Candidate buffer (Section 4.1 "Ordered publication and buffering";
 * Appendix C.1 "Source records and incremental publication").
 *
 * An ordered, append-only buffer of candidate tokens in the target
 * vocabulary.  One producer thread publishes immutable batches of 1..8
 * tokens, each with its provenance record; any number of threads read.
 * A reader takes a snapshot (the published length at that moment) and may
 * read any token below it while later batches are appended; the producer
 * never waits for a reader.  Capacity (tokens) is fixed at creation.
 * These calls touch no GPU state.  Errors: AS2D_EINVAL for null pointers,
 * batch sizes outside 1..8 and reads past the published length;
 * AS2D_ECAPACITY when a batch does not fit; AS2D_ENOMEM.
 */
#define AS2D_MAX_BUDGET 31   /* largest number of candidates per call (max_k <= 31) */

typedef struct as2d_cbuf as2d_cbuf;

typedef struct {
  int64_t first;       /* buffer position of the batch's first token */
  int32_t count;       /* tokens in the batch, 1..8 */
  int32_t source_id;   /* source record (request and audio view) the batch belongs to */
  int32_t producer_id;
  int32_t pad;
  int64_t offset;      /* token offset of the batch within its source sequence */
  int64_t publish_ns;  /* publication time stamp, as given by the producer */
  float confidence;    /* producer confidence, NaN when unavailable */
  int32_t pad2;
} as2d_cbuf_record;

int as2d_cbuf_create(int64_t capacity, as2d_cbuf** out);
int as2d_cbuf_free(as2d_cbuf* buf);
/* Producer only.  *published (optional) receives the new published length. */
int as2d_cbuf_publish(as2d_cbuf* buf, const int32_t* tokens, int32_t n, int32_t source_id, int32_t producer_id,
                      int64_t offset, int64_t publish_ns, float confidence, int64_t* published);
int as2d_cbuf_snapshot(const as2d_cbuf* buf, int64_t* n);
/* Tokens [start, start + n) of the published prefix into out[n] (n = 0
 * reads nothing, at any start >= 0). */
int as2d_cbuf_read(const as2d_cbuf* buf, int64_t start, int32_t n, int32_t* out);
int as2d_cbuf_n_records(const as2d_cbuf* buf, int64_t* n);
int as2d_cbuf_get_record(const as2d_cbuf* buf, int64_t i, as2d_cbuf_record* out);

/*
 * Read cursor and candidate alignment (Section 4.1; Section 4.2 "Candidate
 * alignment"; Appendix C.3 "Candidate alignment"; Figure 4).
 *
 * The cursor moves independently of publication and never changes the
 * buffer.  A plain struct owned by the caller (one per request):
 *   cursor: position of the next candidate to propose;
 *   floor:  lowest position still eligible for realignment (positions below
 *           it were accepted or retired);
 *   radius: bound of the local search (0..64; 8 = one publication batch).
 *
 * as2d_cursor_propose: the ready candidates at the cursor, at most k_max of
 * the first `snapshot` tokens (k = 0 when none is ready: a target-only
 * step).
 *
 * as2d_cursor_update, after a verification call that proposed k
 * candidates from the cursor, accepted `accepted` of them and committed
 * the target token `token` (its correction, or the bonus token after full
 * acceptance), with m = cursor + accepted the position that token stands
 * for.  The target token that follows it is only known after the next
 * call (the token is that call's root), so the rule is read as:
 *   1. accepted > 0: floor = m;
 *   2. if the buffer holds `token` at m (full acceptance whose bonus equals
 *      the next candidate): cursor = floor = m + 1;
 *   3. else the nearest match at distance d = 1..radius, forward (m + d,
 *      below `snapshot`) before backward (m - d, not below floor):
 *      cursor = floor = match + 1.  A forward match skips draft tokens the
 *      target left out; a backward match recovers a token the target
 *      inserted (the candidate it had not reached stays eligible);
 *   4. else cursor = m + 1 (a substitution), floor unchanged.
 * Verification decides every committed token, so the output does not
 * depend on the rule (Appendix C.4, Proposition); the rule decides how
 * many tokens each call commits.
 *
 * as2d_verify_from_buffer: one step of the decoding loop for request req:
 * snapshot, propose at most min(budget, max_commit - 1, AS2D_MAX_BUDGET)
 * candidates, as2d_verify, then as2d_cursor_update against a fresh
 * snapshot.  *k_used (optional) receives the number of candidates
 * verified.  Errors as for as2d_verify; on error the cursor is unchanged.
 */
typedef struct {
  int64_t cursor, floor;
  int32_t radius, pad;
} as2d_read_cursor;

int as2d_cursor_init(as2d_read_cursor* cur, int32_t radius);
int as2d_cursor_propose(const as2d_cbuf* buf, const as2d_read_cursor* cur, int64_t snapshot, int32_t k_max,
                        int32_t* cands, int32_t* k);
int as2d_cursor_update(const as2d_cbuf* buf, as2d_read_cursor* cur, int64_t snapshot, int32_t k, int32_t accepted,
                       int32_t token);
int as2d_verify_from_buffer(as2d_ctx* ctx, int32_t req, const as2d_cbuf* buf, as2d_read_cursor* cur, int32_t budget,
                            int32_t max_commit, as2d_verify_out* out, int32_t* k_used);

/*
 * Target-decoupled decoding with a producer on the same GPU (Section 4.1
 * "Target-decoupled drafting"; the accounting of Appendix D.2, "Overlap,
 * added work, and performance limits").
 *
 * The producer is a drafter model in its own context `drafter` (its own
 * stream), request dreq, prefilled by the caller with capacity for n_draft
 * more positions.  Producer step i is one greedy decode step of the drafter
 * on its own output (as2d_decode_one); the token it publishes for that step
 * is draft[i] (a caller-supplied draft of known quality driven by real
 * drafter compute), in batches of 8 into `buf` (provenance: source 0,
 * producer 1, offset, time since the start of the run).  The verifier
 * (the calling thread) decodes target request treq from the buffer with
 * as2d_verify_from_buffer and `cur` until n_commit tokens are committed;
 * they go to committed[n_commit].
 *   concurrent = 1: the producer runs in its own thread, never waiting for
 *     the verifier, which never waits for it (a target-only step when no
 *     candidate is ready); the run ends when both have stopped.
 *   concurrent = 0: the serial comparator: before each verification the
 *     producer generates whole batches until `budget` candidates past the
 *     cursor are published or the draft is exhausted.
 * Every producer step (kind 0, tokens 1) and verifier call (kind 1, tokens
 * committed) is logged into log[log_cap] as a closed interval in ns from
 * the start of the run (host steady clock, around the synchronous call);
 * *n_log entries, *total_ns the whole run.  Before the producer thread
 * starts, the call captures (under each context's execution mode) every
 * verification graph the two threads will launch: the target's passes of
 * 1..budget + 1 rows and the drafter's one-row step, so no graph is captured
 * while the other thread runs.  `buf` and `cur` must be fresh
 * (nothing published, cursor 0).  A producer error stops the producer only
 * (*producer_rc); the verifier then continues alone.  Errors: as for
 * as2d_verify; AS2D_ECAPACITY when the log is too small.
 */
typedef struct {
  int64_t start_ns, end_ns;
  int32_t kind;    /* 0: producer step, 1: verifier call */
  int32_t tokens;  /* tokens generated (producer) or committed (verifier) */
} as2d_interval;

int as2d_run_decoupled(as2d_ctx* target, int32_t treq, as2d_ctx* drafter, int32_t dreq, const int32_t* draft,
                       int32_t n_draft, int32_t budget, int32_t n_commit, int32_t concurrent, as2d_cbuf* buf,
                       as2d_read_cursor* cur, int32_t* committed, as2d_interval* log, int32_t log_cap,
                       int32_t* n_log, int64_t* total_ns, int32_t* producer_rc);

/* Algorithmic HBM bytes of one forward pass of `rows` rows whose
 * requests hold `kv_keys` attended positions in total per layer
 * (weights streamed once, embedding rows, KV read and append). */
int64_t as2d_step_bytes(const as2d_ctx* ctx, int32_t rows, int64_t kv_keys);

void as2d_free(as2d_ctx* ctx);
const char* as2d_last_error(const as2d_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* AS2D_H */
