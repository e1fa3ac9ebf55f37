// C ABI of the target verification library (include/as2d.h): context and
// request state, weight packing at load time, and the step driver that
// launches the gfx950 kernels of kernels.hip on one HIP stream.
#include "../../include/as2d.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "internal.h"
#include "kernels.h"

using namespace as2d;

namespace {

// Rows of a pass of as2d_verify_static (the direct GEMM path's two row tiles).
constexpr int kStaticRows = kDirectMT * 16;

struct GemmPlan {
  int N = 0, K = 0, KT = 0, pairs = 0, KS = 1, ktps = 0, np = 1, ns = 4;
  int G = 0;  // balanced direct path: workgroups sharing the units (0: one tile per workgroup)
};

struct LayerW {
  uint4 *qkv = nullptr, *o = nullptr, *gu = nullptr, *down = nullptr;
  float *bias = nullptr, *g_attn = nullptr, *g_mlp = nullptr;
};

struct ReqState {
  int active = 0, kv_len = 0, prefix_len = 0, root = -1;
  int last_row_start = 0, last_rows = 0;
  int last_logits = 0;  // logits of the last call are in the device buffer
};

// Device memory one forward pass works in besides the weights and the KV
// cache: activations, split-K and attention partials, arg-max partials,
// counters and the pass's descriptors and results.  A context holds one
// set sized for its largest pass; as2d_verify_static points one into the
// library's static scratch array instead (the launcher takes the set as an
// argument).
struct PassBufs {
  float *x = nullptr, *q = nullptr, *logits = nullptr, *sumsq = nullptr;
  float *amax_val = nullptr, *amax_val2 = nullptr, *row_margin = nullptr;
  float *part = nullptr, *pacc = nullptr, *pml = nullptr;
  int *amax_idx = nullptr, *counters = nullptr, *row_tok = nullptr, *row_bad = nullptr, *fin_counters = nullptr;
  void *xg = nullptr, *attn = nullptr, *hbuf = nullptr;  // activation planes
  long long xg_plane = 0, attn_plane = 0, h_plane = 0;    // offset of the lo plane (bf16), elements
  int part_spans = 0;                                     // span stride of the attention states
  int* attn_cnt = nullptr;                                // finished spans per (request, KV head, row block)
  RowDesc* d_rows = nullptr;
  ReqDesc* d_reqs = nullptr;  // [2 * max_requests]: attention requests, then finish requests
  StepOut* d_out = nullptr;
};

enum Kind { K_EMBED, K_QKV, K_ATTN, K_O, K_GU, K_DOWN, K_LM, K_FINISH, K_STEP, K_COUNT };
const char* kKindNames[K_COUNT] = {"embed", "gemm_qkv", "attention", "gemm_o", "gemm_gate_up",
                                   "gemm_down", "gemm_lm_head", "finish", "step_persistent"};


}  // namespace

struct as2d_ctx {
  as2d_config cfg{};
  bool bf16 = true;
  int es = 2;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  std::string err;
  std::vector<void*> allocs;

  void* embed = nullptr;
  std::vector<LayerW> layers;
  float* g_final = nullptr;
  uint4* lm = nullptr;
  GemmPlan p_qkv, p_o, p_gu, p_down, p_lm;

  float *kc = nullptr, *vc = nullptr;  // float32 KV cache
  long long slot_stride = 0, layer_stride = 0;  // float32 units (a bf16 cache holds twice as many elements)
  int kv_stride = 0;                             // positions per head in the cache: max_kv_len rounded up to 64

  PassBufs b;                 // the context's pass buffers
  float* rope_cs = nullptr;   // rotary table [max_kv_len][head_dim / 2][2]
  void* audio = nullptr;      // audio rows of the prefill being run
  size_t audio_cap = 0;
  int n_blocks_cap = 0;   // 64-key attention blocks of a full slot
  int max_rows = 0;

  RowDesc* h_rows = nullptr;
  ReqDesc* h_reqs = nullptr;
  StepOut* h_out = nullptr;
  int* h_tok = nullptr;
  float* h_margin = nullptr;

  std::vector<ReqState> reqs;
  int keep_logits = 0;

  // execution mode of verification passes (AS2D_EXEC_*) and the captured
  // graphs: (mode, rows, requests, keep_logits) -> executable graph
  int exec_mode = AS2D_EXEC_GRAPH;
  std::map<std::tuple<int, int, int, int>, hipGraphExec_t> graphs;

  // persistent step kernel: per-layer activation buffers and counters
  bool pers_ok = false;
  bool pers_fit = true;          // every balanced plan's grid fits the persistent grid
  int attn_rt = 0;               // row tiles per attention block (0: chosen per pass)
  int pers_grid[3] = {0, 0, 0};  // by M-tile count 1, 2: one workgroup per usable CU
  int pers_sl = 0;               // register-resident slice length of the gate/up plan (0: none)
  float *px = nullptr, *psumsq = nullptr, *pq = nullptr;
  void *pxg = nullptr, *pattn = nullptr, *ph = nullptr;
  int *psplit = nullptr, *pphase = nullptr, *perr = nullptr;
  int split_stride = 0;  // counters per (layer, GEMM)
  int rg_grid = 700;     // staged GEMMs: least grid for row groups of 2-3 tiles
  int n_phase = 0;
  std::map<int, StepLayer*> step_layers;  // by M: device array of per-layer arguments
  int cu_budget = 0;                      // as2d_set_cu_budget (0: all compute units)
  int grid_cus = 0;                       // compute units the grids are sized for
  int h_err = 0;
  long long* ptrace = nullptr;  // persistent-kernel timeline (as2d_set_step_trace)
  int trace_on = 0;

  int timing = 0;
  double t_ms[K_COUNT] = {};
  long long t_n[K_COUNT] = {};
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<int, int>> ev_used;  // (kind, first event index)
};

namespace {

// Message of the last as2d_load_weights failure on this thread (there is
// no context to hold it): as2d_last_error(NULL) returns it.
thread_local std::string t_load_err;

int fail(as2d_ctx* c, int code, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
  }
  return code;
}

#define HIP_TRY(c, expr)                                                                    \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail(c, e_ == hipErrorOutOfMemory ? AS2D_ENOMEM : AS2D_EHIP, "%s: %s (%s:%d)", \
                  #expr, hipGetErrorString(e_), __FILE__, __LINE__);                        \
  } while (0)

template <typename P>
int dalloc(as2d_ctx* c, P** p, size_t bytes) {
  void* v = nullptr;
  hipError_t e = hipMalloc(&v, bytes ? bytes : 16);
  if (e != hipSuccess) return fail(c, AS2D_ENOMEM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
  c->allocs.push_back(v);
  *p = static_cast<P*>(v);
  return AS2D_OK;
}

// Work plan of one matrix.  Wide matrices (at least 1024 tile pairs) give
// each direct-path workgroup two pairs, so one activation fragment feeds
// twice the weights; the others one pair.  Every k-split is summed in 4
// slices (one per wave).  Each compute unit keeps only a bounded amount of
// memory traffic in flight, so the streaming has to reach all of them: the
// k-split count aims at about `target` workgroups per matrix, with at
// least 8 k-steps per split and at most kMaxSplits splits.  The plan
// depends only on the matrix shape, never on the rows of a pass, and the
// pairs per workgroup do not change any sum, so every row is computed
// alike in every pass.
// ks_override > 0 forces the split count (tuning experiments).
GemmPlan make_plan(int N, int K, int KE, int target, int ks_override = 0) {
  GemmPlan p;
  p.N = N;
  p.K = K;
  p.KT = K / KE;
  p.pairs = N / kPairCols;
  p.np = p.pairs >= 1024 ? 2 : 1;
  p.ns = 4;
  int ks = ks_override > 0 ? ks_override : (int)std::lround((double)target / (p.pairs / p.np));
  ks = std::max(1, std::min({ks, std::max(1, p.KT / 8), kMaxSplits}));
  p.ktps = (p.KT + ks - 1) / ks;
  p.KS = (p.KT + p.ktps - 1) / p.ktps;
  return p;
}

// Whether a stream is confined to part of the device by a CU mask
// (hipExtStreamCreateWithCUMask).  Such streams are refused: the first
// concurrent run on masked streams ended in a host segmentation fault whose
// cause has not been found, so the library never runs on one.  A stream
// whose mask cannot be read is taken as unrestricted.
const char* const kRestrictedStream =
    "streams restricted by a CU mask are not supported (use as2d_set_cu_budget to share the device)";
bool stream_restricted(hipStream_t s) {
  int dev = 0, dev_cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&dev_cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || dev_cus < 1)
    return false;
  uint32_t mask[32] = {0};
  const uint32_t words = (uint32_t)((dev_cus + 31) / 32);
  if (words > 32 || hipExtStreamGetCUMask(s, words, mask) != hipSuccess) return false;
  int n = 0;
  for (uint32_t i = 0; i < words; ++i) n += __builtin_popcount(mask[i]);
  return n > 0 && n < dev_cus;
}

// Workgroups of a balanced plan for `cus` compute units: one per CU, at
// most one per unit, and at most kMaxUnits units each.  The split count is
// not touched, so the sums do not change.
void set_grid(GemmPlan& p, int cus) {
  if (!p.G) return;
  const int U = p.pairs * p.KS;
  p.G = std::min(cus, U);
  if ((U + p.G - 1) / p.G > kMaxUnits) p.G = (U + kMaxUnits - 1) / kMaxUnits;
}

// Balanced plan for the direct path (gemm_range kernel): the pairs x KS
// (pair, split) units are shared equally by G = min(compute units, units)
// workgroups.  KS is chosen for the 256 compute units of the MI355X
// whatever the device, so that the sums stay a function of the shape: the
// split count with the least estimated time of the busiest workgroup,
// i.e. units per workgroup x the longest slice of a split (in k-steps),
// plus, with k-splits, `split_cost` k-steps for the fixup phase and
// `per_split` k-steps for each split it reads (measured on the 7B shape:
// 16 and 5 put QKV at 3 splits, O and down at 2, gate/up and the LM head
// at 1, the fastest of the sweep).  Every split needs kWaves k-steps (one
// per slice).  A shape with no such split count keeps the plan `p` (G = 0).
GemmPlan balance_plan(GemmPlan p, int cus, int split_cost, int per_split, int ks_override) {
  constexpr int kNominalCUs = 256;
  int best_ks = 0;
  long long best = 0;
  for (int ks = 1; ks <= kMaxSplits; ++ks) {
    if (ks_override > 0 && ks != ks_override) continue;
    const int ktps = (p.KT + ks - 1) / ks;
    const int kse = (p.KT + ktps - 1) / ktps;
    if (kse != ks || ktps < kWaves || p.KT - (kse - 1) * ktps < kWaves) continue;
    const long long U = (long long)p.pairs * ks;
    const long long G = std::min<long long>(kNominalCUs, U);
    const long long nu = (U + G - 1) / G;
    if (nu > kMaxUnits) continue;
    const long long cost = nu * kWaves * ((ktps + kWaves - 1) / kWaves) + (ks > 1 ? split_cost + per_split * ks : 0);
    if (!best_ks || cost < best) {
      best = cost;
      best_ks = ks;
    }
  }
  if (!best_ks) return p;
  p.np = 1;
  p.ns = kWaves;
  p.ktps = (p.KT + best_ks - 1) / best_ks;
  p.KS = best_ks;
  p.G = 1;
  set_grid(p, cus);
  return p;
}

int env_int(const char* name, int def) {
  const char* v = getenv(name);
  return v && *v ? atoi(v) : def;
}

// Event-bracketed launch accounting (as2d_set_timing).
hipEvent_t ev_get(as2d_ctx* c, size_t i) {
  while (c->ev_pool.size() <= i) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->ev_pool.push_back(e);
  }
  return c->ev_pool[i];
}

struct Timed {
  as2d_ctx* c;
  int kind;
  Timed(as2d_ctx* c_, int k) : c(c_), kind(k) {
    if (c->timing) {
      size_t i = c->ev_used.size() * 2;
      hipEvent_t e = ev_get(c, i);
      ev_get(c, i + 1);
      if (e) hipEventRecord(e, c->stream);
    }
  }
  ~Timed() {
    if (c->timing) {
      size_t i = c->ev_used.size() * 2;
      hipEvent_t e = ev_get(c, i + 1);
      if (e) hipEventRecord(e, c->stream);
      c->ev_used.push_back({kind, (int)i});
    }
  }
};

void timing_collect(as2d_ctx* c) {
  if (!c->timing) return;
  for (auto& u : c->ev_used) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, c->ev_pool[u.second], c->ev_pool[u.second + 1]) == hipSuccess) {
      c->t_ms[u.first] += ms;
      c->t_n[u.first] += 1;
    }
  }
  c->ev_used.clear();
}

int check_req(as2d_ctx* c, int req) {
  if (!c) return AS2D_EINVAL;
  if (req < 0 || req >= c->cfg.max_requests) return fail(c, AS2D_EINVAL, "request id %d out of range", req);
  return AS2D_OK;
}

GemmArgs base_args(as2d_ctx* c, const GemmPlan& pl, const uint4* W, int M, const PassBufs* bp = nullptr) {
  const PassBufs& B = bp ? *bp : c->b;
  GemmArgs a{};
  a.W = W;
  a.N = pl.N;
  a.K = pl.K;
  a.KT = pl.KT;
  a.KS = pl.KS;
  a.ktps = pl.ktps;
  a.np = pl.np;
  a.ns = pl.ns;
  a.G = pl.G;
  a.M = M;
  a.MT = (M + 15) / 16;
  a.rg_grid = c->rg_grid;
  a.sumsq = B.sumsq;
  a.n_norm_pairs = c->cfg.hidden / kPairCols;
  a.a_plane = 0;
  a.eps = c->cfg.rms_eps;
  a.part = B.part;
  a.counters = B.counters;
  a.rows = B.d_rows;
  return a;
}

// Attention score scale: log2(e) / sqrt(d), rounded once to float32 (the
// kernels take base-2 exponentials of the scores).
float attn_scale(int d) { return (float)(1.4426950408889634 / std::sqrt((double)d)); }

// Kernel launches of one forward pass over the rows and requests in the
// device descriptors: n_att attention requests (d_reqs[0..n_att)), n_fin
// finish requests (d_reqs[max_requests..)) covering fin_rows rows;
// with_head = run the LM head and verification; prefill = a prefill pass
// (one request, its rows in order).  max_blocks bounds the
// attention key blocks of any request (it sizes the attention grid).
int launch_pass(as2d_ctx* c, const PassBufs& B, int M, int n_att, int n_fin, int fin_rows, bool with_head,
                int max_blocks, bool prefill) {
  const as2d_config& g = c->cfg;
  hipStream_t s = c->stream;
  const bool bf = c->bf16;
  const int mr = g.max_requests;
  {
    Timed t(c, K_EMBED);
    HIP_TRY(c, launch_embed(bf, B.d_rows, M, c->embed, c->audio, g.hidden, c->layers[0].g_attn, B.x,
                            B.sumsq, B.xg, B.xg_plane, s));
  }
  const int d = g.head_dim;
  for (int l = 0; l < g.n_layers; ++l) {
    const LayerW& w = c->layers[l];
    float* kc = c->kc + (size_t)l * c->layer_stride;
    float* vc = c->vc + (size_t)l * c->layer_stride;
    const float* g_next = l + 1 < g.n_layers ? c->layers[l + 1].g_attn : c->g_final;
    {
      GemmArgs a = base_args(c, c->p_qkv, w.qkv, M, &B);
      a.A = B.xg;
      a.a_plane = B.xg_plane;
      a.bias = w.bias;
      a.q_out = B.q;
      a.k_cache = kc;
      a.v_cache = vc;
      a.slot_stride = c->slot_stride;
      a.kv_cap = c->kv_stride;
      a.n_q = g.n_q_heads;
      a.n_kv = g.n_kv_heads;
      a.head_dim = d;
      a.rope_cs = c->rope_cs;
      Timed t(c, K_QKV);
      HIP_TRY(c, launch_gemm(bf, A_NORM, EPI_QKV, a, s));
    }
    {
      AttnArgs a{};
      a.q = B.q;
      a.k_cache = kc;
      a.v_cache = vc;
      a.slot_stride = c->slot_stride;
      a.kv_cap = c->kv_stride;
      a.rows = B.d_rows;
      a.reqs = B.d_reqs;
      a.n_q = g.n_q_heads;
      a.n_kv = g.n_kv_heads;
      a.head_dim = d;
      a.scale = attn_scale(d);
      a.pacc = B.pacc;
      a.pml = B.pml;
      a.part_spans = B.part_spans;
      // caches of up to 16 spans: the span kernel merges (no second launch)
      a.merge_last = B.part_spans <= 16;
      a.attn_cnt = B.attn_cnt;
      a.out = B.attn;
      a.out_plane = B.attn_plane;
      a.M = M;
      a.attn_rt = c->attn_rt;
      a.cus = c->grid_cus;
      Timed t(c, K_ATTN);
      HIP_TRY(c, launch_attention(bf, a, n_att, max_blocks, prefill, s));
    }
    {
      GemmArgs a = base_args(c, c->p_o, w.o, M, &B);
      a.A = B.attn;
      a.a_plane = B.attn_plane;
      a.x = B.x;
      a.x_out = B.x;
      a.sumsq_out = B.sumsq;
      a.gain_next = w.g_mlp;
      a.out = B.xg;
      a.out_plane = B.xg_plane;
      Timed t(c, K_O);
      HIP_TRY(c, launch_gemm(bf, A_PLAIN, EPI_RESID, a, s));
    }
    {
      GemmArgs a = base_args(c, c->p_gu, w.gu, M, &B);
      a.A = B.xg;
      a.a_plane = B.xg_plane;
      a.out = B.hbuf;
      a.out_plane = B.h_plane;
      Timed t(c, K_GU);
      HIP_TRY(c, launch_gemm(bf, A_NORM, EPI_SWIGLU, a, s));
    }
    {
      GemmArgs a = base_args(c, c->p_down, w.down, M, &B);
      a.A = B.hbuf;
      a.a_plane = B.h_plane;
      a.x = B.x;
      a.x_out = B.x;
      a.sumsq_out = B.sumsq;
      a.gain_next = g_next;
      a.out = B.xg;
      a.out_plane = B.xg_plane;
      Timed t(c, K_DOWN);
      HIP_TRY(c, launch_gemm(bf, A_PLAIN, EPI_DOWN, a, s));
    }
  }
  if (with_head) {
    {
      GemmArgs a = base_args(c, c->p_lm, c->lm, M, &B);
      a.A = B.xg;
      a.a_plane = B.xg_plane;
      a.logits = c->keep_logits ? B.logits : nullptr;
      a.amax_val = B.amax_val;
      a.amax_val2 = B.amax_val2;
      a.amax_idx = B.amax_idx;
      Timed t(c, K_LM);
      HIP_TRY(c, launch_gemm(bf, A_NORM, EPI_ARGMAX, a, s));
    }
    {
      Timed t(c, K_FINISH);
      HIP_TRY(c, launch_finish(B.d_rows, B.d_reqs + mr, n_fin, fin_rows, B.amax_val, B.amax_val2, B.amax_idx,
                               g.vocab / kPairCols, B.row_tok, B.row_bad, B.row_margin, B.fin_counters,
                               B.d_out, s));
    }
  }
  return AS2D_OK;
}

// Per-layer arguments of the persistent step kernel for passes of M rows
// (device array, built once per M).
StepLayer* step_layers_for(as2d_ctx* c, int M) {
  auto it = c->step_layers.find(M);
  if (it != c->step_layers.end()) return it->second;
  const as2d_config& g = c->cfg;
  const int H = g.hidden, F = g.ffn, d = g.head_dim, nq = g.n_q_heads, nkv = g.n_kv_heads;
  const long long R = kStepRows;
  const size_t xs = (size_t)R * H;                        // floats of one x / planes of one xg
  const size_t ss = (size_t)(H / kPairCols) * kMaxRows;   // sum-of-squares partials
  const size_t qs = (size_t)R * nq * d;
  auto xg = [&](int i) { return (void*)((char*)c->pxg + i * xs * 4); };
  std::vector<StepLayer> v(g.n_layers);
  for (int l = 0; l < g.n_layers; ++l) {
    const LayerW& w = c->layers[l];
    StepLayer& s = v[l];
    float* kc = c->kc + (size_t)l * c->layer_stride;
    float* vc = c->vc + (size_t)l * c->layer_stride;
    int* cnt = c->psplit + (size_t)(4 * l) * c->split_stride;
    s.qkv = base_args(c, c->p_qkv, w.qkv, M);
    s.qkv.A = xg(2 * l);
    s.qkv.a_plane = c->bf16 ? (long long)xs : 0;
    s.qkv.sumsq = c->psumsq + (2 * l) * ss;
    s.qkv.counters = cnt;
    s.qkv.bias = w.bias;
    s.qkv.q_out = c->pq + l * qs;
    s.qkv.k_cache = kc;
    s.qkv.v_cache = vc;
    s.qkv.slot_stride = c->slot_stride;
    s.qkv.kv_cap = c->kv_stride;
    s.qkv.n_q = nq;
    s.qkv.n_kv = nkv;
    s.qkv.head_dim = d;
    s.qkv.rope_cs = c->rope_cs;

    AttnArgs& a = s.attn;
    a = AttnArgs{};
    a.q = c->pq + l * qs;
    a.k_cache = kc;
    a.v_cache = vc;
    a.slot_stride = c->slot_stride;
    a.kv_cap = c->kv_stride;
    a.rows = c->b.d_rows;
    a.reqs = c->b.d_reqs;
    a.n_q = nq;
    a.n_kv = nkv;
    a.head_dim = d;
    a.scale = attn_scale(d);
    a.pacc = c->b.pacc;
    a.pml = c->b.pml;
    a.part_spans = c->b.part_spans;
    a.out = (char*)c->pattn + l * qs * 4;
    a.out_plane = c->bf16 ? (long long)qs : 0;
    a.M = M;

    s.o = base_args(c, c->p_o, w.o, M);
    s.o.A = a.out;
    s.o.a_plane = a.out_plane;
    s.o.counters = cnt + c->split_stride;
    s.o.x = c->px + (2 * l) * xs;
    s.o.x_out = c->px + (2 * l + 1) * xs;
    s.o.sumsq_out = c->psumsq + (2 * l + 1) * ss;
    s.o.gain_next = w.g_mlp;
    s.o.out = xg(2 * l + 1);
    s.o.out_plane = c->bf16 ? (long long)xs : 0;

    s.gu = base_args(c, c->p_gu, w.gu, M);
    s.gu.A = xg(2 * l + 1);
    s.gu.a_plane = c->bf16 ? (long long)xs : 0;
    s.gu.sumsq = c->psumsq + (2 * l + 1) * ss;
    s.gu.counters = cnt + 2 * c->split_stride;
    s.gu.out = (char*)c->ph + (size_t)l * R * F * 4;
    s.gu.out_plane = c->bf16 ? R * F : 0;

    s.down = base_args(c, c->p_down, w.down, M);
    s.down.A = s.gu.out;
    s.down.a_plane = s.gu.out_plane;
    s.down.counters = cnt + 3 * c->split_stride;
    s.down.x = c->px + (2 * l + 1) * xs;
    s.down.x_out = c->px + (2 * l + 2) * xs;
    s.down.sumsq_out = c->psumsq + (2 * l + 2) * ss;
    s.down.gain_next = l + 1 < g.n_layers ? c->layers[l + 1].g_attn : c->g_final;
    s.down.out = xg(2 * l + 2);
    s.down.out_plane = c->bf16 ? (long long)xs : 0;
  }
  StepLayer* dv = nullptr;
  if (hipMalloc(&dv, sizeof(StepLayer) * g.n_layers) != hipSuccess) return nullptr;
  c->allocs.push_back(dv);
  if (hipMemcpy(dv, v.data(), sizeof(StepLayer) * g.n_layers, hipMemcpyHostToDevice) != hipSuccess) return nullptr;
  c->step_layers[M] = dv;
  return dv;
}

// Launches of one verification pass through the persistent step kernel.
int launch_persistent(as2d_ctx* c, int M, int n_att, int n_fin, int fin_rows) {
  const as2d_config& g = c->cfg;
  StepLayer* layers = step_layers_for(c, M);
  if (!layers) return fail(c, AS2D_ENOMEM, "persistent step arguments");
  const int L = g.n_layers, H = g.hidden;
  const size_t xs = (size_t)kStepRows * H;
  const size_t ss = (size_t)(H / kPairCols) * kMaxRows;
  StepArgs a{};
  a.layers = layers;
  a.n_layers = L;
  a.lm = base_args(c, c->p_lm, c->lm, M);
  a.lm.A = (char*)c->pxg + 2 * L * xs * 4;
  a.lm.a_plane = c->bf16 ? (long long)xs : 0;
  a.lm.sumsq = c->psumsq + 2 * L * ss;
  a.lm.counters = c->psplit + (size_t)(4 * L) * c->split_stride;
  a.lm.logits = c->keep_logits ? c->b.logits : nullptr;
  a.lm.amax_val = c->b.amax_val;
  a.lm.amax_val2 = c->b.amax_val2;
  a.lm.amax_idx = c->b.amax_idx;
  a.M = M;
  a.rows = c->b.d_rows;
  a.embed = c->embed;
  a.audio = c->audio;
  a.hidden = H;
  a.gain0 = c->layers[0].g_attn;
  a.x0 = c->px;
  a.sumsq0 = c->psumsq;
  a.xg0 = c->pxg;
  a.xg0_plane = c->bf16 ? (long long)xs : 0;
  a.reqs = c->b.d_reqs;
  a.n_reqs = n_att;
  a.n_q = g.n_q_heads;
  a.n_kv = g.n_kv_heads;
  a.fin_reqs = c->b.d_reqs + g.max_requests;
  a.n_fin = n_fin;
  a.fin_rows = fin_rows;
  a.row_tok = c->b.row_tok;
  a.row_bad = c->b.row_bad;
  a.row_margin = c->b.row_margin;
  a.out = c->b.d_out;
  // completion signals of a GEMM phase: one per workgroup of a balanced
  // plan, else one per tile pair
  const int grid = c->pers_grid[(M + 15) / 16];
  for (const GemmPlan* p : {&c->p_qkv, &c->p_o, &c->p_gu, &c->p_down, &c->p_lm})
    if (p->G < 1 || p->G > grid)
      return fail(c, AS2D_ESTATE, "persistent step: plan grid %d outside [1, %d]", p->G, grid);
  {
    GemmArgs probe[5] = {base_args(c, c->p_qkv, nullptr, M), base_args(c, c->p_o, nullptr, M),
                         base_args(c, c->p_gu, nullptr, M), base_args(c, c->p_down, nullptr, M), a.lm};
    for (const GemmArgs& p : probe)
      if (!range_plan_ok(p)) return fail(c, AS2D_ESTATE, "persistent step: plan outside the balanced path");
  }
  a.done_qkv = c->p_qkv.G;
  a.done_o = c->p_o.G;
  a.done_gu = c->p_gu.G;
  a.done_down = c->p_down.G;
  a.done_lm = c->p_lm.G;
  a.phase_cnt = c->pphase;
  a.err = c->perr;
  a.spin_limit = env_int("AS2D_SPIN_LIMIT", 1 << 21);
  a.trace = c->trace_on ? c->ptrace : nullptr;
  const int MT = (M + 15) / 16;
  Timed t(c, K_STEP);
  HIP_TRY(c, launch_step(c->bf16, MT, g.head_dim, c->pers_sl, a, grid, c->n_phase, c->stream));
  return AS2D_OK;
}

// The executable graph of a verification pass of M rows over n_att
// requests (fin_rows rows verified), captured on first use.  Kernel
// arguments hold only pointers and sizes (the row and request descriptors
// are read from device memory when the graph runs) and the attention grid
// covers the slot capacity, so one graph serves every pass of that shape.
int graph_for(as2d_ctx* c, int M, int n_att, int n_fin, int fin_rows, bool persistent, hipGraphExec_t* out) {
  const auto key = std::make_tuple((int)persistent, M, n_att, c->keep_logits);
  auto it = c->graphs.find(key);
  if (it == c->graphs.end()) {
    if (c->graphs.size() >= 64) {
      for (auto& kv : c->graphs) hipGraphExecDestroy(kv.second);
      c->graphs.clear();
    }
    hipGraph_t gr = nullptr;
    HIP_TRY(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal));
    int rc = persistent ? launch_persistent(c, M, n_att, n_fin, fin_rows)
                        : launch_pass(c, c->b, M, n_att, n_fin, fin_rows, true, c->n_blocks_cap, false);
    hipError_t e = hipStreamEndCapture(c->stream, &gr);
    if (rc) {
      if (gr) hipGraphDestroy(gr);
      return rc;
    }
    if (e != hipSuccess) return fail(c, AS2D_EHIP, "graph capture: %s", hipGetErrorString(e));
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, gr, nullptr, nullptr, 0);
    hipGraphDestroy(gr);
    if (e != hipSuccess) return fail(c, AS2D_EHIP, "graph instantiate: %s", hipGetErrorString(e));
    it = c->graphs.emplace(key, ex).first;
  }
  *out = it->second;
  return AS2D_OK;
}

// One forward pass over the rows and requests in h_rows / h_reqs (see
// launch_pass).  Verification passes run as a captured HIP graph, one per
// (rows, requests, keep_logits); the attention grid then covers the slot
// capacity so that the graph stays valid as the cache grows.
int run_forward(as2d_ctx* c, int M, int n_att, int n_fin, bool with_head, bool verify_call = false) {
  const as2d_config& g = c->cfg;
  hipStream_t s = c->stream;
  const int mr = g.max_requests;
  int fin_rows = 0;
  for (int r = 0; r < n_fin; ++r) fin_rows += c->h_reqs[mr + r].W;
  HIP_TRY(c, hipMemcpyAsync(c->b.d_rows, c->h_rows, sizeof(RowDesc) * M, hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(c->b.d_reqs, c->h_reqs, sizeof(ReqDesc) * 2 * mr, hipMemcpyHostToDevice, s));
  int max_blocks = 1;
  for (int r = 0; r < n_att; ++r) {
    const int nk = c->h_reqs[r].L0 + c->h_reqs[r].W;
    max_blocks = std::max(max_blocks, (nk + kAttnBlock - 1) / kAttnBlock);
  }
  if (max_blocks > c->n_blocks_cap) return fail(c, AS2D_ECAPACITY, "attention blocks %d > %d", max_blocks, c->n_blocks_cap);
  const bool verify_pass = verify_call && with_head && n_fin == n_att;
  const bool persistent = verify_pass && c->exec_mode == AS2D_EXEC_PERSISTENT && c->pers_ok && c->pers_fit && M <= kStepRows;
  const bool graph = verify_pass && c->exec_mode != AS2D_EXEC_EAGER && !c->timing;
  if (persistent && !step_layers_for(c, M)) return fail(c, AS2D_ENOMEM, "persistent step arguments");
  if (graph) {
    hipGraphExec_t ex = nullptr;
    int rc = graph_for(c, M, n_att, n_fin, fin_rows, persistent, &ex);
    if (rc) return rc;
    HIP_TRY(c, hipGraphLaunch(ex, s));
  } else {
    int rc = persistent ? launch_persistent(c, M, n_att, n_fin, fin_rows)
                        : launch_pass(c, c->b, M, n_att, n_fin, fin_rows, with_head, max_blocks, !verify_call);
    if (rc) return rc;
  }
  if (persistent) HIP_TRY(c, hipMemcpyAsync(&c->h_err, c->perr, sizeof(int), hipMemcpyDeviceToHost, s));
  if (with_head) {
    HIP_TRY(c, hipMemcpyAsync(c->h_out, c->b.d_out, sizeof(StepOut) * n_fin, hipMemcpyDeviceToHost, s));
    HIP_TRY(c, hipMemcpyAsync(c->h_tok, c->b.row_tok, sizeof(int) * M, hipMemcpyDeviceToHost, s));
    HIP_TRY(c, hipMemcpyAsync(c->h_margin, c->b.row_margin, sizeof(float) * M, hipMemcpyDeviceToHost, s));
  }
  HIP_TRY(c, hipStreamSynchronize(s));
  timing_collect(c);
  if (persistent && c->h_err) {
    c->h_err = 0;
    HIP_TRY(c, hipMemset(c->perr, 0, sizeof(int)));
    return fail(c, AS2D_EHIP, "persistent step kernel: a wait timed out (workgroups not co-resident?)");
  }
  return AS2D_OK;
}

}  // namespace

int as2d_prepare_graphs(as2d_ctx* c, int32_t max_rows) {
  if (!c || max_rows < 1) return AS2D_EINVAL;
  if (c->exec_mode == AS2D_EXEC_EAGER || c->timing) return AS2D_OK;   // no graphs in these modes
  max_rows = std::min(max_rows, c->cfg.max_k + 1);
  for (int M = 1; M <= max_rows; ++M) {
    const bool persistent = c->exec_mode == AS2D_EXEC_PERSISTENT && c->pers_ok && c->pers_fit && M <= kStepRows;
    if (persistent && !step_layers_for(c, M)) return fail(c, AS2D_ENOMEM, "persistent step arguments");
    hipGraphExec_t ex = nullptr;
    const int rc = graph_for(c, M, 1, 1, M, persistent, &ex);
    if (rc) return rc;
  }
  return AS2D_OK;
}

namespace {

int upload_matrix(as2d_ctx* c, void* tmp, const void* host, size_t rows, size_t cols) {
  HIP_TRY(c, hipMemcpyAsync(tmp, host, rows * cols * c->es, hipMemcpyHostToDevice, c->stream));
  return AS2D_OK;
}

int pack(as2d_ctx* c, uint4** out, const void* tmp, int N, int K, int map, int arg) {
  int rc = dalloc(c, out, (size_t)N * K * c->es);
  if (rc) return rc;
  HIP_TRY(c, launch_pack(c->bf16, tmp, *out, N, K, map, arg, c->stream));
  return AS2D_OK;
}

// Forget everything captured from the current launch parameters: the
// verification graphs (grids are kernel launch parameters) and the
// persistent kernel's per-layer argument arrays (they hold each plan's
// grid).  Called after a grid change, with the stream idle.
void drop_launch_state(as2d_ctx* c) {
  for (auto& kv : c->graphs) hipGraphExecDestroy(kv.second);
  c->graphs.clear();
  for (auto& kv : c->step_layers) {
    auto it = std::find(c->allocs.begin(), c->allocs.end(), (void*)kv.second);
    if (it != c->allocs.end()) c->allocs.erase(it);
    hipFree(kv.second);
  }
  c->step_layers.clear();
}

// Balanced GEMM grids and the persistent kernel's grid for `cus` compute
// units (0: the whole device).  Split counts, and so every result, do not
// depend on it.
int set_grids(as2d_ctx* c, int cus) {
  int dev = 0, dev_cus = 0;
  HIP_TRY(c, hipGetDevice(&dev));
  HIP_TRY(c, hipDeviceGetAttribute(&dev_cus, hipDeviceAttributeMultiprocessorCount, dev));
  const int n = cus > 0 ? std::min(cus, dev_cus) : dev_cus;
  c->grid_cus = n;
  // a plan whose units would exceed kMaxUnits per workgroup on n keeps a
  // wider grid; the persistent kernel, one workgroup per CU of the budget,
  // then cannot hold that phase and verification passes use graphs
  int widest = 0;
  for (GemmPlan* p : {&c->p_qkv, &c->p_o, &c->p_gu, &c->p_down, &c->p_lm}) {
    set_grid(*p, n);
    widest = std::max(widest, p->G);
  }
  c->pers_fit = widest <= n;
  if (c->pers_ok)
    for (int mt = 1; mt <= 2; ++mt) c->pers_grid[mt] = n;
  return AS2D_OK;
}

// Checks the arguments of a verification call of n requests (at most
// max_rows rows in all) and writes its row and request descriptors into
// h_rows / h_reqs; *M receives the row count.
int assemble_verify(as2d_ctx* c, int n, const int32_t* reqs, const int32_t* cands, const int32_t* ks,
                    const as2d_verify_out* outs, int max_rows, int* M_out) {
  if (!c) return AS2D_EINVAL;
  const as2d_config& g = c->cfg;
  if (n < 1 || n > g.max_requests || !reqs || !ks || !outs) return fail(c, AS2D_EINVAL, "verify: bad arguments");
  int M = 0, off = 0;
  const int mr = g.max_requests;
  for (int r = 0; r < n; ++r) {
    int rc = check_req(c, reqs[r]);
    if (rc) return rc;
    for (int q = 0; q < r; ++q)
      if (reqs[q] == reqs[r]) return fail(c, AS2D_EINVAL, "verify: request %d listed twice", reqs[r]);
    const ReqState& st = c->reqs[reqs[r]];
    if (!st.active) return fail(c, AS2D_ESTATE, "verify: request %d has not been prefilled", reqs[r]);
    const int k = ks[r];
    if (k < 0 || k > g.max_k) return fail(c, AS2D_EINVAL, "verify: k=%d outside [0, %d]", k, g.max_k);
    if (k && !cands) return fail(c, AS2D_EINVAL, "verify: null candidates");
    for (int i = 0; i < k; ++i)
      if (cands[off + i] < 0 || cands[off + i] >= g.vocab)
        return fail(c, AS2D_EINVAL, "verify: candidate id %d out of range", cands[off + i]);
    if (st.kv_len + k + 1 > g.max_kv_len)
      return fail(c, AS2D_ECAPACITY, "verify: request %d needs %d positions > %d", reqs[r], st.kv_len + k + 1, g.max_kv_len);
    M += k + 1;
    off += k;
  }
  if (M > max_rows) return fail(c, AS2D_EINVAL, "verify: %d rows exceed %d", M, max_rows);
  int row = 0;
  off = 0;
  for (int r = 0; r < n; ++r) {
    const ReqState& st = c->reqs[reqs[r]];
    const int k = ks[r];
    for (int i = 0; i <= k; ++i) {
      RowDesc rd{};
      rd.token = i == 0 ? st.root : cands[off + i - 1];
      rd.src = 0;
      rd.pos = st.kv_len + i;
      rd.slot = reqs[r];
      rd.cmp = i < k ? cands[off + i] : -1;
      c->h_rows[row + i] = rd;
    }
    c->h_reqs[r] = ReqDesc{row, k + 1, st.kv_len, reqs[r]};
    c->h_reqs[mr + r] = c->h_reqs[r];
    row += k + 1;
    off += k;
  }
  *M_out = M;
  return AS2D_OK;
}

// Commits the outcome in h_out of the verification call assembled by
// assemble_verify: accepted rows stay in the cache, the correction becomes
// the root; a request with non-finite logits keeps its state.
int commit_verify(as2d_ctx* c, int n, const int32_t* reqs, const int32_t* ks, as2d_verify_out* outs) {
  const as2d_config& g = c->cfg;
  int n_bad = 0, first_bad = -1;
  for (int r = 0; r < n; ++r) {
    ReqState& st = c->reqs[reqs[r]];
    const StepOut& o = c->h_out[r];
    st.last_row_start = c->h_reqs[r].row_start;
    st.last_rows = ks[r] + 1;
    st.last_logits = c->keep_logits;
    if (o.nan_flag) {
      // no token can be chosen: this request keeps its state
      if (!n_bad++) first_bad = reqs[r];
      outs[r].accepted_len = -1;
      outs[r].correction_token = -1;
      outs[r].kv_len = st.kv_len;
      outs[r].committed = st.kv_len - st.prefix_len;
      continue;
    }
    st.kv_len += o.accepted + 1;
    st.root = o.correction;
    outs[r].accepted_len = o.accepted;
    outs[r].correction_token = o.correction;
    outs[r].kv_len = st.kv_len;
    outs[r].committed = st.kv_len - st.prefix_len;
  }
  // other requests' last-call rows are no longer in the device buffers
  for (int q = 0; q < g.max_requests; ++q) {
    bool in = false;
    for (int r = 0; r < n; ++r) in |= reqs[r] == q;
    if (!in) c->reqs[q].last_logits = 0, c->reqs[q].last_rows = 0;
  }
  if (n_bad) return fail(c, AS2D_ENUMERIC, "verify: non-finite logits in %d request(s) (first: %d)", n_bad, first_bad);
  return AS2D_OK;
}

// Split-K counters a pass may use: one per workgroup tile (at most one per
// tile pair on the direct path; on the staged path one per (group of
// kPairsS pairs, row group), at most kMaxMTiles row groups).
int split_counter_count(const as2d_ctx* c) {
  int n = 0;
  for (const GemmPlan* p : {&c->p_qkv, &c->p_o, &c->p_gu, &c->p_down, &c->p_lm})
    n = std::max({n, p->pairs, (p->pairs / kPairsS) * kMaxMTiles});
  return n;
}

// Pass buffers for passes of up to kStaticRows rows over n_blocks key
// blocks, laid out from `base` (256-byte aligned pieces); returns the
// bytes they span.  The logits (an output the caller reads with
// as2d_get_logits) stay in the context.
size_t static_layout(const as2d_ctx* c, int n_blocks, char* base, PassBufs* S) {
  const as2d_config& g = c->cfg;
  const size_t R = kStaticRows, H = g.hidden, F = g.ffn, V = g.vocab, QD = (size_t)g.n_q_heads * g.head_dim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base + off;
    off += (bytes + 255) / 256 * 256;
    return (void*)p;
  };
  size_t part = 0;
  for (const GemmPlan* p : {&c->p_qkv, &c->p_o, &c->p_gu, &c->p_down, &c->p_lm})
    if (p->KS > 1) part = std::max(part, (size_t)p->KS * R * p->N);
  S->d_rows = (RowDesc*)take(sizeof(RowDesc) * R);
  S->d_reqs = (ReqDesc*)take(sizeof(ReqDesc) * 2 * g.max_requests);
  S->d_out = (StepOut*)take(sizeof(StepOut) * g.max_requests);
  S->x = (float*)take(R * H * 4);
  S->q = (float*)take(R * QD * 4);
  S->xg = take(R * H * 4);
  S->attn = take(R * QD * 4);
  S->hbuf = take(R * F * 4);
  if (c->bf16) {
    S->xg_plane = (long long)(R * H);
    S->attn_plane = (long long)(R * QD);
    S->h_plane = (long long)(R * F);
  }
  S->logits = c->b.logits;
  S->sumsq = (float*)take((H / kPairCols) * R * 4);
  S->amax_val = (float*)take((V / kPairCols) * R * 4);
  S->amax_val2 = (float*)take((V / kPairCols) * R * 4);
  S->amax_idx = (int*)take((V / kPairCols) * R * 4);
  S->row_tok = (int*)take(R * 4);
  S->row_bad = (int*)take(R * 4);
  S->row_margin = (float*)take(R * 4);
  S->fin_counters = (int*)take((size_t)g.max_requests * 4);
  S->part = (float*)take(part * 4);
  S->counters = (int*)take((size_t)split_counter_count(c) * 4);
  S->part_spans = (int)((n_blocks + kAttnSpan - 1) / kAttnSpan);
  const size_t spans = (n_blocks + kAttnSpan - 1) / kAttnSpan;
  S->pacc = (float*)take(spans * R * QD * 4);
  S->pml = (float*)take(spans * R * g.n_q_heads * 2 * 4);
  S->attn_cnt = (int*)take((size_t)g.max_requests * g.n_q_heads * 2 * 4);
  return off;
}

}  // namespace

// ===========================================================================
// C ABI

extern "C" {

const char* as2d_last_error(const as2d_ctx* c) {
  if (c) return c->err.c_str();
  return t_load_err.empty() ? "null context" : t_load_err.c_str();
}

void as2d_free(as2d_ctx* c) {
  if (!c) return;
  if (c->stream) hipStreamSynchronize(c->stream);
  for (void* p : c->allocs) hipFree(p);
  if (c->h_rows) hipHostFree(c->h_rows);
  if (c->h_reqs) hipHostFree(c->h_reqs);
  if (c->h_out) hipHostFree(c->h_out);
  if (c->h_tok) hipHostFree(c->h_tok);
  if (c->h_margin) hipHostFree(c->h_margin);
  for (hipEvent_t e : c->ev_pool) hipEventDestroy(e);
  for (auto& kv : c->graphs) hipGraphExecDestroy(kv.second);
  if (c->own_stream && c->stream) hipStreamDestroy(c->stream);
  delete c;
}

int as2d_load_weights(const as2d_config* cfg, const void* const* host, int32_t n_tensors,
                      void* hip_stream, as2d_ctx** out) {
  if (!cfg || !host || !out) return AS2D_EINVAL;
  *out = nullptr;
  const as2d_config g = *cfg;
  t_load_err.clear();
  auto c = new as2d_ctx();
  // every failure below frees the context; its message stays readable
  // through as2d_last_error(NULL)
  auto give_up = [&](int code) {
    t_load_err = c->err.empty() ? "as2d_load_weights failed" : c->err;
    as2d_free(c);
    return code;
  };
  auto bad = [&](const char* msg) {
    c->err = std::string("as2d_load_weights: ") + msg;
    return give_up(AS2D_EINVAL);
  };
  if (g.n_layers < 1 || g.hidden % 128 || g.ffn % 64 || g.vocab % 128 || g.vocab <= 0)
    return bad("shape: need n_layers >= 1, hidden % 128 == 0, ffn % 64 == 0, vocab % 128 == 0");
  if (g.head_dim != 64 && g.head_dim != 128) return bad("head_dim must be 64 or 128");
  if (g.n_q_heads < 1 || g.n_kv_heads < 1 || g.n_q_heads % g.n_kv_heads)
    return bad("n_q_heads must be a positive multiple of n_kv_heads");
  if (((g.n_q_heads + 2 * g.n_kv_heads) * g.head_dim) % 128 || (g.n_q_heads * g.head_dim) % 128)
    return bad("attention widths must be multiples of 128");
  if (g.dtype != AS2D_F32 && g.dtype != AS2D_BF16) return bad("dtype must be AS2D_F32 or AS2D_BF16");
  if (g.max_requests < 1 || g.max_kv_len < 2 || g.max_kv_len > kMaxBlocks * kAttnBlock || g.max_k < 0 ||
      g.max_k > 31)
    return bad("capacity: max_requests >= 1, 2 <= max_kv_len <= 32768, 0 <= max_k <= 31");
  if (g.hidden > 8192) return bad("hidden must be <= 8192");
  if (!(g.rms_eps >= 0.f) || !(g.rope_theta > 0.f)) return bad("rms_eps >= 0 and rope_theta > 0 required");
  const int per_layer = g.qkv_bias ? 12 : 9;
  if (n_tensors != 1 + per_layer * g.n_layers + 2) return bad("wrong tensor count for this config");
  for (int i = 0; i < n_tensors; ++i)
    if (!host[i]) return bad("null tensor pointer");

  c->cfg = g;
  c->bf16 = g.dtype == AS2D_BF16;
  c->es = c->bf16 ? 2 : 4;
  const int KE = c->bf16 ? 32 : 16;
  const int H = g.hidden, F = g.ffn, V = g.vocab, d = g.head_dim;
  const int nq = g.n_q_heads, nkv = g.n_kv_heads;
  const int qkv_n = (nq + 2 * nkv) * d;
  int rc;
  // inside `run` errors return their code; the caller frees the context
#define CK(x)                      \
  do {                             \
    if ((rc = (x)) != 0) return rc; \
  } while (0)

  if (hip_stream) {
    c->stream = (hipStream_t)hip_stream;
  } else {
    if (hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking) != hipSuccess) {
      c->err = "as2d_load_weights: hipStreamCreateWithFlags failed";
      return give_up(AS2D_EHIP);
    }
    c->own_stream = true;
  }
  if (stream_restricted(c->stream)) return bad(kRestrictedStream);
  if (H % KE || (nq * d) % KE || F % KE) return bad("inner dimensions must be multiples of the k-step");

  // GEMM plans: k-splits depend on the matrix shape only
  const int target = env_int("AS2D_TARGET_WGS", 256);
  const int ks_qkv = env_int("AS2D_KS_QKV", 0), ks_o = env_int("AS2D_KS_O", 0), ks_gu = env_int("AS2D_KS_GU", 0);
  const int ks_down = env_int("AS2D_KS_DOWN", 0), ks_lm = env_int("AS2D_KS_LM", 0);
  c->rg_grid = env_int("AS2D_RG_GRID", 700);
  c->p_qkv = make_plan(qkv_n, H, KE, target, ks_qkv);
  c->p_o = make_plan(H, nq * d, KE, target, ks_o);
  c->p_gu = make_plan(2 * F, H, KE, target, ks_gu);
  c->p_down = make_plan(H, F, KE, target, ks_down);
  c->p_lm = make_plan(V, H, KE, target, ks_lm);
  // balanced direct path, per matrix (bits: QKV 1, O 2, gate/up 4, down 8, LM head 16)
  const int bal = env_int("AS2D_BALANCED", 31);
  if (bal) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                hipSuccess || cus < 1) {
      fail(c, AS2D_EHIP, "as2d_load_weights: device query");
      return give_up(AS2D_EHIP);
    }
    const int sc = env_int("AS2D_SPLIT_COST", 16), ps = env_int("AS2D_SPLIT_COST_PER", 5);
    if (bal & 1) c->p_qkv = balance_plan(c->p_qkv, cus, sc, ps, ks_qkv);
    if (bal & 2) c->p_o = balance_plan(c->p_o, cus, sc, ps, ks_o);
    if (bal & 4) c->p_gu = balance_plan(c->p_gu, cus, sc, ps, ks_gu);
    if (bal & 8) c->p_down = balance_plan(c->p_down, cus, sc, ps, ks_down);
    if (bal & 16) c->p_lm = balance_plan(c->p_lm, cus, sc, ps, ks_lm);
  }

  // temporary device buffer for raw matrices before packing (largest matrix)
  size_t tmp_elems = std::max({(size_t)V * H, (size_t)qkv_n * H, (size_t)2 * F * H, (size_t)H * F});
  void* tmp = nullptr;
  if (hipMalloc(&tmp, tmp_elems * c->es) != hipSuccess) {
    fail(c, AS2D_ENOMEM, "as2d_load_weights: staging buffer");
    return give_up(AS2D_ENOMEM);
  }
  auto run = [&]() -> int {
    int ti = 0;
    int rc = 0;
    CK(dalloc(c, &c->embed, (size_t)V * H * c->es));
    HIP_TRY(c, hipMemcpyAsync(c->embed, host[ti++], (size_t)V * H * c->es, hipMemcpyHostToDevice, c->stream));
    c->layers.resize(g.n_layers);
    for (int l = 0; l < g.n_layers; ++l) {
      LayerW& w = c->layers[l];
      CK(dalloc(c, &w.g_attn, H * 4));
      HIP_TRY(c, hipMemcpyAsync(w.g_attn, host[ti++], H * 4, hipMemcpyHostToDevice, c->stream));
      // q, k, v rows stacked into one [qkv_n][H] matrix
      char* t = (char*)tmp;
      HIP_TRY(c, hipMemcpyAsync(t, host[ti++], (size_t)nq * d * H * c->es, hipMemcpyHostToDevice, c->stream));
      t += (size_t)nq * d * H * c->es;
      HIP_TRY(c, hipMemcpyAsync(t, host[ti++], (size_t)nkv * d * H * c->es, hipMemcpyHostToDevice, c->stream));
      t += (size_t)nkv * d * H * c->es;
      HIP_TRY(c, hipMemcpyAsync(t, host[ti++], (size_t)nkv * d * H * c->es, hipMemcpyHostToDevice, c->stream));
      CK(pack(c, &w.qkv, tmp, qkv_n, H, PACK_ROPE_PAIRS, d));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
      if (g.qkv_bias) {
        CK(dalloc(c, &w.bias, qkv_n * 4));
        HIP_TRY(c, hipMemcpyAsync(w.bias, host[ti++], nq * d * 4, hipMemcpyHostToDevice, c->stream));
        HIP_TRY(c, hipMemcpyAsync(w.bias + nq * d, host[ti++], nkv * d * 4, hipMemcpyHostToDevice, c->stream));
        HIP_TRY(c, hipMemcpyAsync(w.bias + (nq + nkv) * d, host[ti++], nkv * d * 4, hipMemcpyHostToDevice, c->stream));
      }
      CK(upload_matrix(c, tmp, host[ti++], H, nq * d));
      CK(pack(c, &w.o, tmp, H, nq * d, PACK_IDENTITY, 0));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
      CK(dalloc(c, &w.g_mlp, H * 4));
      HIP_TRY(c, hipMemcpyAsync(w.g_mlp, host[ti++], H * 4, hipMemcpyHostToDevice, c->stream));
      CK(upload_matrix(c, tmp, host[ti++], F, H));
      CK(upload_matrix(c, (char*)tmp + (size_t)F * H * c->es, host[ti++], F, H));
      CK(pack(c, &w.gu, tmp, 2 * F, H, PACK_GATE_UP, F));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
      CK(upload_matrix(c, tmp, host[ti++], H, F));
      CK(pack(c, &w.down, tmp, H, F, PACK_IDENTITY, 0));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
    }
    CK(dalloc(c, &c->g_final, H * 4));
    HIP_TRY(c, hipMemcpyAsync(c->g_final, host[ti++], H * 4, hipMemcpyHostToDevice, c->stream));
    CK(upload_matrix(c, tmp, host[ti++], V, H));
    CK(pack(c, &c->lm, tmp, V, H, PACK_IDENTITY, 0));
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    return AS2D_OK;
  };
  rc = run();
  hipFree(tmp);
  if (rc == 0) rc = [&]() -> int {
    int rc = 0;

  // KV cache: [slot][layer][kv_head][pos][d]
  c->kv_stride = (g.max_kv_len + 63) / 64 * 64;
  c->layer_stride = (long long)nkv * c->kv_stride * d;
  c->slot_stride = c->layer_stride * g.n_layers;
  const size_t kv_bytes = (size_t)c->slot_stride * g.max_requests * sizeof(float);
  CK(dalloc(c, &c->kc, kv_bytes));
  CK(dalloc(c, &c->vc, kv_bytes));

  // activations and scratch, sized for the largest pass
  c->max_rows = kMaxRows;   // rows per pass (prefill chunks, fused batches)
  const int MR = kMaxRows;
  c->n_blocks_cap = (g.max_kv_len + kAttnBlock - 1) / kAttnBlock;
  CK(dalloc(c, &c->b.x, (size_t)MR * H * 4));
  CK(dalloc(c, &c->b.q, (size_t)MR * nq * d * 4));
  // activation planes: two bf16 planes or one float32 plane, 4 bytes per element either way
  CK(dalloc(c, &c->b.xg, (size_t)MR * H * 4));
  CK(dalloc(c, &c->b.attn, (size_t)MR * nq * d * 4));
  CK(dalloc(c, &c->b.hbuf, (size_t)MR * F * 4));
  if (c->bf16) {
    c->b.xg_plane = (long long)MR * H;
    c->b.attn_plane = (long long)MR * nq * d;
    c->b.h_plane = (long long)MR * F;
  }
  CK(dalloc(c, &c->b.logits, (size_t)MR * V * 4));
  CK(dalloc(c, &c->b.sumsq, (size_t)(H / kPairCols) * MR * 4));
  CK(dalloc(c, &c->b.amax_val, (size_t)(V / kPairCols) * MR * 4));
  CK(dalloc(c, &c->b.amax_val2, (size_t)(V / kPairCols) * MR * 4));
  CK(dalloc(c, &c->b.row_margin, (size_t)MR * 4));
  CK(dalloc(c, &c->b.amax_idx, (size_t)(V / kPairCols) * MR * 4));
  CK(dalloc(c, &c->b.row_tok, (size_t)MR * 4));
  CK(dalloc(c, &c->b.row_bad, (size_t)MR * 4));
  CK(dalloc(c, &c->b.fin_counters, (size_t)g.max_requests * 4));
  HIP_TRY(c, hipMemsetAsync(c->b.fin_counters, 0, (size_t)g.max_requests * 4, c->stream));
  size_t part_elems = 0;
  for (const GemmPlan* p : {&c->p_qkv, &c->p_o, &c->p_gu, &c->p_down, &c->p_lm})
    if (p->KS > 1) part_elems = std::max(part_elems, (size_t)p->KS * MR * p->N);
  CK(dalloc(c, &c->b.part, part_elems * 4));
  const int n_cnt = split_counter_count(c);
  CK(dalloc(c, &c->b.counters, (size_t)n_cnt * 4));
  HIP_TRY(c, hipMemsetAsync(c->b.counters, 0, (size_t)n_cnt * 4, c->stream));
  HIP_TRY(c, prepare_kernels());
  {
    // the static scratch of as2d_verify_static: its address on this device
    void* p = nullptr;
    size_t n = 0;
    HIP_TRY(c, static_scratch(&p, &n));
  }
  // persistent step kernel (verification passes of up to 32 rows; every
  // GEMM on a balanced plan)
  bool all_balanced = true;
  for (const GemmPlan* p : {&c->p_qkv, &c->p_o, &c->p_gu, &c->p_down, &c->p_lm}) all_balanced &= p->G > 0;
  if (all_balanced && env_int("AS2D_PERSISTENT", 1)) {
    int dev = 0, cus = 0, occ1 = 0, occ2 = 0;
    HIP_TRY(c, hipGetDevice(&dev));
    HIP_TRY(c, hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    c->pers_sl = step_ra_slice(c->bf16, c->p_gu.KS, c->p_gu.KT);
    HIP_TRY(c, step_occupancy(c->bf16, 1, d, H, c->pers_sl, &occ1));
    HIP_TRY(c, step_occupancy(c->bf16, 2, d, H, 0, &occ2));
    const int L = g.n_layers;
    const long long R = kStepRows;
    if (occ1 > 0 && occ2 > 0) {
      c->pers_grid[1] = cus;
      c->pers_grid[2] = cus;
      CK(dalloc(c, &c->px, (size_t)(2 * L + 1) * R * H * 4));
      CK(dalloc(c, &c->pxg, (size_t)(2 * L + 1) * R * H * 4));
      CK(dalloc(c, &c->psumsq, (size_t)(2 * L + 1) * (H / kPairCols) * kMaxRows * 4));
      CK(dalloc(c, &c->pq, (size_t)L * R * nq * d * 4));
      CK(dalloc(c, &c->pattn, (size_t)L * R * nq * d * 4));
      CK(dalloc(c, &c->ph, (size_t)L * R * F * 4));
      c->split_stride = std::max({c->p_qkv.pairs, c->p_o.pairs, c->p_gu.pairs, c->p_down.pairs,
                                  c->p_lm.pairs});
      const size_t n_split = (size_t)(4 * L + 1) * c->split_stride;
      CK(dalloc(c, &c->psplit, n_split * 4));
      HIP_TRY(c, hipMemsetAsync(c->psplit, 0, n_split * 4, c->stream));
      c->n_phase = 3 + 6 * L;
      CK(dalloc(c, &c->pphase, (size_t)c->n_phase * 4));
      CK(dalloc(c, &c->perr, 4));
      HIP_TRY(c, hipMemsetAsync(c->perr, 0, 4, c->stream));
      c->pers_ok = true;
    }
  }
  c->b.part_spans = (int)((c->n_blocks_cap + kAttnSpan - 1) / kAttnSpan);
  const size_t spans_cap = (c->n_blocks_cap + kAttnSpan - 1) / kAttnSpan;
  CK(dalloc(c, &c->b.pacc, spans_cap * MR * nq * d * 4));
  CK(dalloc(c, &c->b.pml, spans_cap * MR * nq * 2 * 4));
  CK(dalloc(c, &c->b.attn_cnt, (size_t)g.max_requests * nq * 2 * 4));
  HIP_TRY(c, hipMemsetAsync(c->b.attn_cnt, 0, (size_t)g.max_requests * nq * 2 * 4, c->stream));
  CK(dalloc(c, &c->b.d_rows, sizeof(RowDesc) * MR));
  CK(dalloc(c, &c->b.d_reqs, sizeof(ReqDesc) * 2 * g.max_requests));
  CK(dalloc(c, &c->b.d_out, sizeof(StepOut) * g.max_requests));

  // rotary table, evaluated in double precision: [pos][i] -> (cos, sin)
  {
    const int half = d / 2;
    std::vector<float> cs((size_t)g.max_kv_len * half * 2);
    for (int pos = 0; pos < g.max_kv_len; ++pos)
      for (int i = 0; i < half; ++i) {
        const double ang = (double)pos * std::pow((double)g.rope_theta, -2.0 * i / d);
        cs[((size_t)pos * half + i) * 2] = (float)std::cos(ang);
        cs[((size_t)pos * half + i) * 2 + 1] = (float)std::sin(ang);
      }
    CK(dalloc(c, &c->rope_cs, cs.size() * 4));
    HIP_TRY(c, hipMemcpy(c->rope_cs, cs.data(), cs.size() * 4, hipMemcpyHostToDevice));
  }
  if (hipHostMalloc((void**)&c->h_rows, sizeof(RowDesc) * MR, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->h_reqs, sizeof(ReqDesc) * 2 * g.max_requests, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->h_out, sizeof(StepOut) * g.max_requests, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->h_tok, sizeof(int) * MR, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->h_margin, sizeof(float) * MR, 0) != hipSuccess) {
    return fail(c, AS2D_ENOMEM, "pinned host buffers");
  }
  memset(c->h_reqs, 0, sizeof(ReqDesc) * 2 * g.max_requests);
  c->reqs.assign(g.max_requests, ReqState());
  c->exec_mode = env_int("AS2D_EXEC_MODE", AS2D_EXEC_GRAPH);
  c->attn_rt = env_int("AS2D_ATTN_RT", 0);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return AS2D_OK;
  }();
  if (rc) return give_up(rc);
  *out = c;
  return AS2D_OK;
#undef CK
}

int as2d_prefill_kv(as2d_ctx* c, int32_t req, const void* audio, int32_t n_audio,
                    const int32_t* instr, int32_t n_instr, int32_t* first_token, int32_t* kv_len) {
  int rc = check_req(c, req);
  if (rc) return rc;
  const as2d_config& g = c->cfg;
  if (n_audio < 0 || n_instr < 0 || n_audio + n_instr < 1 || (n_audio && !audio) || (n_instr && !instr) ||
      !first_token || !kv_len)
    return fail(c, AS2D_EINVAL, "prefill: bad arguments");
  const int total = n_audio + n_instr;
  if (total > g.max_kv_len) return fail(c, AS2D_ECAPACITY, "prefill: %d rows > max_kv_len %d", total, g.max_kv_len);
  for (int i = 0; i < n_instr; ++i)
    if (instr[i] < 0 || instr[i] >= g.vocab) return fail(c, AS2D_EINVAL, "prefill: token id %d out of range", instr[i]);
  ReqState& st = c->reqs[req];
  st = ReqState();
  if (n_audio) {
    const size_t bytes = (size_t)n_audio * g.hidden * c->es;
    if (bytes > c->audio_cap) {
      if (c->audio) {
        HIP_TRY(c, hipStreamSynchronize(c->stream));
        auto it = std::find(c->allocs.begin(), c->allocs.end(), c->audio);
        if (it != c->allocs.end()) c->allocs.erase(it);
        hipFree(c->audio);
        c->audio = nullptr;
        c->audio_cap = 0;
      }
      if ((rc = dalloc(c, &c->audio, bytes))) return rc;
      c->audio_cap = bytes;
    }
    HIP_TRY(c, hipMemcpyAsync(c->audio, audio, bytes, hipMemcpyHostToDevice, c->stream));
  }
  const int chunk = c->max_rows;
  const int mr = g.max_requests;
  for (int r0 = 0; r0 < total; r0 += chunk) {
    const int M = std::min(chunk, total - r0);
    for (int i = 0; i < M; ++i) {
      const int p = r0 + i;
      RowDesc rd{};
      rd.token = p < n_audio ? -1 : instr[p - n_audio];
      rd.src = p < n_audio ? p : 0;
      rd.pos = p;
      rd.slot = req;
      rd.cmp = -1;
      c->h_rows[i] = rd;
    }
    c->h_reqs[0] = ReqDesc{0, M, r0, req};
    const bool last = r0 + M == total;
    c->h_reqs[mr] = ReqDesc{M - 1, 1, r0 + M - 1, req};
    if ((rc = run_forward(c, M, 1, 1, last))) return rc;
    if (last) {
      if (c->h_out[0].nan_flag) return fail(c, AS2D_ENUMERIC, "prefill: non-finite logits");
      st.root = c->h_out[0].correction;
      st.last_row_start = M - 1;
      st.last_rows = 1;
      st.last_logits = c->keep_logits;
    }
  }
  st.active = 1;
  st.kv_len = st.prefix_len = total;
  // the prefill's passes overwrote the shared logits and row-token buffers
  for (int q = 0; q < g.max_requests; ++q)
    if (q != req) c->reqs[q].last_logits = 0, c->reqs[q].last_rows = 0;
  *first_token = st.root;
  *kv_len = total;
  return AS2D_OK;
}

int as2d_verify_batch(as2d_ctx* c, int32_t n, const int32_t* reqs, const int32_t* cands,
                      const int32_t* ks, as2d_verify_out* outs) {
  int M = 0;
  int rc = assemble_verify(c, n, reqs, cands, ks, outs, kMaxRows, &M);
  if (rc) return rc;
  if ((rc = run_forward(c, M, n, n, true, true))) return rc;
  return commit_verify(c, n, reqs, ks, outs);
}

int as2d_verify_static(as2d_ctx* c, int32_t req, const int32_t* cands, int32_t k, as2d_verify_out* out) {
  int M = 0;
  int rc = assemble_verify(c, 1, &req, cands, &k, out, kStaticRows, &M);
  if (rc) return rc;
  const as2d_config& g = c->cfg;
  const int mr = g.max_requests;
  const int n_blocks = (c->h_reqs[0].L0 + M + kAttnBlock - 1) / kAttnBlock;
  void* base = nullptr;
  size_t cap = 0;
  HIP_TRY(c, static_scratch(&base, &cap));
  PassBufs S;
  const size_t need = static_layout(c, n_blocks, (char*)base, &S);
  if (need > cap)
    return fail(c, AS2D_ECAPACITY, "verify_static: the pass needs %zu bytes of static scratch, %zu available (%d keys)",
                need, cap, c->h_reqs[0].L0 + M);
  hipStream_t s = c->stream;
  HIP_TRY(c, hipMemcpyAsync(S.d_rows, c->h_rows, sizeof(RowDesc) * M, hipMemcpyHostToDevice, s));
  HIP_TRY(c, hipMemcpyAsync(S.d_reqs, c->h_reqs, sizeof(ReqDesc) * 2 * mr, hipMemcpyHostToDevice, s));
  // the array keeps the last call's contents: counters must start at zero
  HIP_TRY(c, launch_fill_zero(S.counters, split_counter_count(c), s));
  HIP_TRY(c, launch_fill_zero(S.fin_counters, mr, s));
  HIP_TRY(c, launch_fill_zero(S.attn_cnt, mr * g.n_q_heads * 2, s));
  const int timing = c->timing;   // no event bracketing here (events are created on first use)
  c->timing = 0;
  rc = launch_pass(c, S, M, 1, 1, M, true, n_blocks, false);
  c->timing = timing;
  if (rc) return rc;
  HIP_TRY(c, hipMemcpyAsync(c->h_out, S.d_out, sizeof(StepOut), hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipMemcpyAsync(c->h_tok, S.row_tok, sizeof(int) * M, hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipMemcpyAsync(c->h_margin, S.row_margin, sizeof(float) * M, hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipStreamSynchronize(s));
  return commit_verify(c, 1, &req, &k, out);
}

int as2d_verify(as2d_ctx* c, int32_t req, const int32_t* cands, int32_t k, as2d_verify_out* out) {
  return as2d_verify_batch(c, 1, &req, cands, &k, out);
}

int as2d_decode_one(as2d_ctx* c, int32_t req, as2d_verify_out* out) {
  const int32_t k = 0;
  return as2d_verify_batch(c, 1, &req, nullptr, &k, out);
}

int as2d_set_keep_logits(as2d_ctx* c, int32_t on) {
  if (!c) return AS2D_EINVAL;
  c->keep_logits = on ? 1 : 0;
  return AS2D_OK;
}

int as2d_get_logits(as2d_ctx* c, int32_t req, float* host, int32_t max_rows, int32_t* n_rows) {
  int rc = check_req(c, req);
  if (rc) return rc;
  const ReqState& st = c->reqs[req];
  if (!host || !n_rows) return fail(c, AS2D_EINVAL, "get_logits: null pointer");
  if (!st.last_logits || !st.last_rows) return fail(c, AS2D_ESTATE, "get_logits: no logits kept for request %d", req);
  if (max_rows < st.last_rows) return fail(c, AS2D_EINVAL, "get_logits: need %d rows", st.last_rows);
  HIP_TRY(c, hipMemcpy(host, c->b.logits + (size_t)st.last_row_start * c->cfg.vocab,
                       (size_t)st.last_rows * c->cfg.vocab * 4, hipMemcpyDeviceToHost));
  *n_rows = st.last_rows;
  return AS2D_OK;
}

int as2d_get_row_tokens(as2d_ctx* c, int32_t req, int32_t* host, int32_t max_rows, int32_t* n_rows) {
  int rc = check_req(c, req);
  if (rc) return rc;
  const ReqState& st = c->reqs[req];
  if (!host || !n_rows) return fail(c, AS2D_EINVAL, "get_row_tokens: null pointer");
  if (!st.last_rows) return fail(c, AS2D_ESTATE, "get_row_tokens: no rows for request %d", req);
  if (max_rows < st.last_rows) return fail(c, AS2D_EINVAL, "get_row_tokens: need %d rows", st.last_rows);
  memcpy(host, c->h_tok + st.last_row_start, sizeof(int) * st.last_rows);
  *n_rows = st.last_rows;
  return AS2D_OK;
}

int as2d_get_row_margins(as2d_ctx* c, int32_t req, float* host, int32_t max_rows, int32_t* n_rows) {
  int rc = check_req(c, req);
  if (rc) return rc;
  const ReqState& st = c->reqs[req];
  if (!host || !n_rows) return fail(c, AS2D_EINVAL, "get_row_margins: null pointer");
  if (!st.last_rows) return fail(c, AS2D_ESTATE, "get_row_margins: no rows for request %d", req);
  if (max_rows < st.last_rows) return fail(c, AS2D_EINVAL, "get_row_margins: need %d rows", st.last_rows);
  memcpy(host, c->h_margin + st.last_row_start, sizeof(float) * st.last_rows);
  *n_rows = st.last_rows;
  return AS2D_OK;
}

int as2d_rollback(as2d_ctx* c, int32_t req, int32_t kv_len, int32_t root) {
  int rc = check_req(c, req);
  if (rc) return rc;
  ReqState& st = c->reqs[req];
  if (!st.active) return fail(c, AS2D_ESTATE, "rollback: request %d has not been prefilled", req);
  if (kv_len < st.prefix_len || kv_len > st.kv_len)
    return fail(c, AS2D_EINVAL, "rollback: kv_len %d outside [%d, %d]", kv_len, st.prefix_len, st.kv_len);
  if (root < 0 || root >= c->cfg.vocab) return fail(c, AS2D_EINVAL, "rollback: root id out of range");
  st.kv_len = kv_len;
  st.root = root;
  st.last_rows = 0;
  st.last_logits = 0;
  return AS2D_OK;
}

int as2d_get_state(as2d_ctx* c, int32_t req, int32_t* kv_len, int32_t* root, int32_t* committed) {
  int rc = check_req(c, req);
  if (rc) return rc;
  const ReqState& st = c->reqs[req];
  if (!st.active) return fail(c, AS2D_ESTATE, "request %d has not been prefilled", req);
  if (kv_len) *kv_len = st.kv_len;
  if (root) *root = st.root;
  if (committed) *committed = st.kv_len - st.prefix_len;
  return AS2D_OK;
}

int as2d_read_kv(as2d_ctx* c, int32_t req, int32_t layer, void* host_k, void* host_v, int32_t n_tok) {
  int rc = check_req(c, req);
  if (rc) return rc;
  const as2d_config& g = c->cfg;
  if (layer < 0 || layer >= g.n_layers || n_tok < 0 || n_tok > g.max_kv_len || !host_k || !host_v)
    return fail(c, AS2D_EINVAL, "read_kv: bad arguments");
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  const size_t d = (size_t)g.head_dim, cap = (size_t)c->kv_stride;
  float* ok = static_cast<float*>(host_k);
  float* ov = static_cast<float*>(host_v);
  // one head's cache region: cap * d floats of K (positions, then dimensions:
  // bf16 (hi, lo) rows or float32 rows) and of V (dimensions, then positions:
  // bf16 (hi, lo) planes or one float32 plane)
  std::vector<float> kbuf(cap * d), vbuf(cap * d);
  auto hi16 = [](const float* base, size_t i) {
    uint16_t h;
    memcpy(&h, reinterpret_cast<const char*>(base) + 2 * i, 2);
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
  };
  for (int h = 0; h < g.n_kv_heads; ++h) {
    const size_t src = (size_t)req * c->slot_stride + (size_t)layer * c->layer_stride + (size_t)h * cap * d;
    HIP_TRY(c, hipMemcpy(kbuf.data(), c->kc + src, cap * d * 4, hipMemcpyDeviceToHost));
    HIP_TRY(c, hipMemcpy(vbuf.data(), c->vc + src, cap * d * 4, hipMemcpyDeviceToHost));
    for (size_t t = 0; t < (size_t)n_tok; ++t)
      for (size_t j = 0; j < d; ++j) {
        float kv, vv;
        if (c->bf16) {
          kv = hi16(kbuf.data(), t * 2 * d + j) + hi16(kbuf.data(), t * 2 * d + d + j);
          vv = hi16(vbuf.data(), v_elem((int)t, 0, (int)j, (int)d, true)) +
               hi16(vbuf.data(), v_elem((int)t, 1, (int)j, (int)d, true));
        } else {
          kv = kbuf[t * d + j];
          vv = vbuf[v_elem((int)t, 0, (int)j, (int)d, false)];
        }
        ok[((size_t)h * n_tok + t) * d + j] = kv;
        ov[((size_t)h * n_tok + t) * d + j] = vv;
      }
  }
  return AS2D_OK;
}

int as2d_set_stream(as2d_ctx* c, void* hip_stream) {
  if (!c) return AS2D_EINVAL;
  if (hip_stream && stream_restricted((hipStream_t)hip_stream)) return fail(c, AS2D_EINVAL, "set_stream: %s", kRestrictedStream);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  drop_launch_state(c);
  if (c->own_stream) {
    hipStreamDestroy(c->stream);
    c->own_stream = false;
    c->stream = nullptr;
  }
  if (hip_stream) {
    c->stream = (hipStream_t)hip_stream;
  } else {
    HIP_TRY(c, hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking));
    c->own_stream = true;
  }
  return set_grids(c, c->cu_budget);
}

int as2d_set_cu_budget(as2d_ctx* c, int32_t cus) {
  if (!c || cus < 0) return AS2D_EINVAL;
  int dev = 0, dev_cus = 0;
  HIP_TRY(c, hipGetDevice(&dev));
  HIP_TRY(c, hipDeviceGetAttribute(&dev_cus, hipDeviceAttributeMultiprocessorCount, dev));
  if (cus > dev_cus) return fail(c, AS2D_EINVAL, "cu budget %d > %d compute units", cus, dev_cus);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  drop_launch_state(c);
  c->cu_budget = cus;
  return set_grids(c, cus);
}

int as2d_release_request(as2d_ctx* c, int32_t req) {
  int rc = check_req(c, req);
  if (rc) return rc;
  c->reqs[req] = ReqState();
  return AS2D_OK;
}

int as2d_set_exec_mode(as2d_ctx* c, int32_t mode) {
  if (!c) return AS2D_EINVAL;
  if (mode < AS2D_EXEC_EAGER || mode > AS2D_EXEC_PERSISTENT) return fail(c, AS2D_EINVAL, "unknown exec mode %d", mode);
  c->exec_mode = mode;
  return AS2D_OK;
}

int as2d_get_exec_info(as2d_ctx* c, int32_t* mode, int32_t* persistent_grid) {
  if (!c) return AS2D_EINVAL;
  if (mode) *mode = c->exec_mode;
  if (persistent_grid) *persistent_grid = c->pers_ok && c->pers_fit ? c->pers_grid[1] : 0;
  return AS2D_OK;
}

int as2d_set_step_trace(as2d_ctx* c, int32_t on) {
  if (!c) return AS2D_EINVAL;
  if (!c->pers_ok) return fail(c, AS2D_ESTATE, "no persistent step kernel on this device");
  if (on && !c->ptrace) {
    // sized for the whole device: a later compute-unit budget can widen the grid
    int dev = 0, dev_cus = 0;
    HIP_TRY(c, hipGetDevice(&dev));
    HIP_TRY(c, hipDeviceGetAttribute(&dev_cus, hipDeviceAttributeMultiprocessorCount, dev));
    const size_t n = (size_t)std::max({c->pers_grid[1], c->pers_grid[2], dev_cus}) * c->n_phase * 3;
    int rc = dalloc(c, &c->ptrace, n * sizeof(long long));
    if (rc) return rc;
    HIP_TRY(c, hipMemset(c->ptrace, 0, n * sizeof(long long)));
  }
  c->trace_on = on ? 1 : 0;
  for (auto& kv : c->graphs) hipGraphExecDestroy(kv.second);  // the trace pointer is a kernel argument
  c->graphs.clear();
  return AS2D_OK;
}

int as2d_step_trace_read(as2d_ctx* c, int64_t* host, int64_t max, int32_t* grid, int32_t* n_phase) {
  if (!c || !host || !grid || !n_phase) return AS2D_EINVAL;
  if (!c->ptrace) return fail(c, AS2D_ESTATE, "step trace not enabled");
  const int G = std::max(c->pers_grid[1], c->pers_grid[2]);
  const int64_t n = (int64_t)G * c->n_phase * 3;
  if (max < n) return fail(c, AS2D_EINVAL, "need %lld entries", (long long)n);
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  HIP_TRY(c, hipMemcpy(host, c->ptrace, n * sizeof(long long), hipMemcpyDeviceToHost));
  *grid = G;
  *n_phase = c->n_phase;
  return AS2D_OK;
}

int as2d_set_timing(as2d_ctx* c, int32_t on) {
  if (!c) return AS2D_EINVAL;
  c->timing = on ? 1 : 0;
  return AS2D_OK;
}

int as2d_timing_reset(as2d_ctx* c) {
  if (!c) return AS2D_EINVAL;
  for (int k = 0; k < K_COUNT; ++k) c->t_ms[k] = 0, c->t_n[k] = 0;
  return AS2D_OK;
}

int as2d_timing_read(as2d_ctx* c, char* names, double* total_ms, int64_t* counts, int32_t max) {
  if (!c || !names || !total_ms || !counts) return AS2D_EINVAL;
  const int n = std::min<int>(max, K_COUNT);
  for (int k = 0; k < n; ++k) {
    snprintf(names + 32 * k, 32, "%s", kKindNames[k]);
    total_ms[k] = c->t_ms[k];
    counts[k] = c->t_n[k];
  }
  return n;
}

int as2d_time_gemm(as2d_ctx* c, int32_t which, int32_t rows, int32_t reps, double* avg_us) {
  if (!c || !avg_us || which < 0 || which > 4 || rows < 1 || rows > kMaxRows || reps < 1)
    return c ? fail(c, AS2D_EINVAL, "time_gemm: bad arguments") : AS2D_EINVAL;
  const as2d_config& g = c->cfg;
  hipStream_t s = c->stream;
  // rows describe positions 0..rows-1 of slot 0: only the QKV epilogue reads
  // them (cache rows it overwrites are in bounds; their contents are garbage)
  for (int i = 0; i < rows; ++i) c->h_rows[i] = RowDesc{0, 0, std::min(i, g.max_kv_len - 1), 0, -1, {0, 0, 0}};
  HIP_TRY(c, hipMemcpyAsync(c->b.d_rows, c->h_rows, sizeof(RowDesc) * rows, hipMemcpyHostToDevice, s));
  hipEvent_t e0 = ev_get(c, 1000), e1 = ev_get(c, 1001);
  if (!e0 || !e1) return fail(c, AS2D_EHIP, "time_gemm: events");
  auto launch = [&](int l) -> int {
    const LayerW& w = c->layers[l];
    GemmArgs a;
    int am = A_NORM, epi = EPI_QKV;
    switch (which) {
      case 0:
        a = base_args(c, c->p_qkv, w.qkv, rows);
        a.A = c->b.xg; a.a_plane = c->b.xg_plane; a.bias = w.bias; a.q_out = c->b.q;
        a.k_cache = c->kc + (size_t)l * c->layer_stride; a.v_cache = c->vc + (size_t)l * c->layer_stride;
        a.slot_stride = c->slot_stride; a.kv_cap = c->kv_stride; a.n_q = g.n_q_heads;
        a.n_kv = g.n_kv_heads; a.head_dim = g.head_dim; a.rope_cs = c->rope_cs;
        break;
      case 1:
        a = base_args(c, c->p_o, w.o, rows);
        a.A = c->b.attn; a.a_plane = c->b.attn_plane; a.x = c->b.x; a.x_out = c->b.x; a.sumsq_out = c->b.sumsq;
        a.gain_next = w.g_mlp; a.out = c->b.xg; a.out_plane = c->b.xg_plane;
        am = A_PLAIN; epi = EPI_RESID;
        break;
      case 2:
        a = base_args(c, c->p_gu, w.gu, rows);
        a.A = c->b.xg; a.a_plane = c->b.xg_plane; a.out = c->b.hbuf; a.out_plane = c->b.h_plane;
        epi = EPI_SWIGLU;
        break;
      case 3:
        a = base_args(c, c->p_down, w.down, rows);
        a.A = c->b.hbuf; a.a_plane = c->b.h_plane; a.x = c->b.x; a.x_out = c->b.x; a.sumsq_out = c->b.sumsq;
        a.gain_next = w.g_attn; a.out = c->b.xg; a.out_plane = c->b.xg_plane;
        am = A_PLAIN; epi = EPI_DOWN;
        break;
      default:
        a = base_args(c, c->p_lm, c->lm, rows);
        a.A = c->b.xg; a.a_plane = c->b.xg_plane; a.amax_val = c->b.amax_val; a.amax_val2 = c->b.amax_val2;
        a.amax_idx = c->b.amax_idx;
        epi = EPI_ARGMAX;
    }
    HIP_TRY(c, launch_gemm(c->bf16, am, epi, a, s));
    return AS2D_OK;
  };
  int rc = launch(0);  // warm-up
  if (rc) return rc;
  HIP_TRY(c, hipEventRecord(e0, s));
  for (int i = 0; i < reps; ++i)
    if ((rc = launch(which == 4 ? 0 : i % g.n_layers))) return rc;
  HIP_TRY(c, hipEventRecord(e1, s));
  HIP_TRY(c, hipEventSynchronize(e1));
  float ms = 0.f;
  HIP_TRY(c, hipEventElapsedTime(&ms, e0, e1));
  *avg_us = ms * 1e3 / reps;
  return AS2D_OK;
}

int as2d_stream_bandwidth(as2d_ctx* c, int64_t bytes, int32_t reps, double* gbps) {
  constexpr int64_t kUnit = 64ll << 20;
  if (!c || !gbps || bytes < kUnit || reps < 1)
    return c ? fail(c, AS2D_EINVAL, "stream_bandwidth: bad arguments") : AS2D_EINVAL;
  bytes = bytes / kUnit * kUnit;
  hipStream_t s = c->stream;
  int dev = 0, cus = 0;
  HIP_TRY(c, hipGetDevice(&dev));
  HIP_TRY(c, hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  void* buf = nullptr;
  unsigned* out = nullptr;
  if (hipMalloc(&buf, (size_t)bytes) != hipSuccess) return fail(c, AS2D_ENOMEM, "stream_bandwidth: %lld bytes", (long long)bytes);
  int rc = [&]() -> int {
    HIP_TRY(c, hipMalloc(&out, (size_t)cus * 4 * sizeof(unsigned)));
    HIP_TRY(c, hipMemsetAsync(buf, 0, (size_t)bytes, s));
    // one workgroup per compute unit; the segments must be whole 8 KiB runs per wave
    int grid = cus;
    while (grid > 1 && (bytes / 16) % ((int64_t)grid * 4 * 512)) --grid;
    hipEvent_t e0 = ev_get(c, 1002), e1 = ev_get(c, 1003);
    if (!e0 || !e1) return fail(c, AS2D_EHIP, "stream_bandwidth: events");
    HIP_TRY(c, launch_stream_read((const uint4*)buf, bytes / 16, grid, out, s));   // warm-up
    HIP_TRY(c, hipEventRecord(e0, s));
    for (int i = 0; i < reps; ++i) HIP_TRY(c, launch_stream_read((const uint4*)buf, bytes / 16, grid, out, s));
    HIP_TRY(c, hipEventRecord(e1, s));
    HIP_TRY(c, hipEventSynchronize(e1));
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, e0, e1));
    *gbps = (double)bytes * reps / (ms * 1e-3) / 1e9;
    return AS2D_OK;
  }();
  hipStreamSynchronize(s);
  if (out) hipFree(out);
  hipFree(buf);
  return rc;
}

int64_t as2d_step_bytes(const as2d_ctx* c, int32_t rows, int64_t kv_keys) {
  if (!c) return -1;
  const as2d_config& g = c->cfg;
  const int64_t H = g.hidden, F = g.ffn, V = g.vocab, d = g.head_dim;
  const int64_t nq = g.n_q_heads, nkv = g.n_kv_heads;
  const int64_t per_layer = H * (nq + 2 * nkv) * d + nq * d * H + 3 * H * F;
  int64_t b = c->es * (g.n_layers * per_layer + V * H);  // weights, streamed once
  b += c->es * rows * H;                                 // embedding rows
  b += 4 * g.n_layers * 2 * nkv * d * (kv_keys + rows);  // float32 KV read + append
  return b;
}

}  // extern "C"
