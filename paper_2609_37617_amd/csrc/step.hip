// Persistent step kernel: one launch runs a whole verification pass
// (embedding, every decoder layer, LM head and greedy verification) for up
// to 32 rows.
//
// All workgroups are resident at once (one per compute unit).  The pass
// is a sequence of phases; a phase's work is split over the workgroups,
// which walk the phases in order.  A GEMM phase runs the balanced units of
// its plan: a workgroup first issues its weight loads (weights do not
// depend on activations), then waits until the producing phase's
// completion counter reaches its target, so weight streaming continues
// across phase boundaries instead of stopping at a kernel boundary.
// Attention spans (attn.h) are dealt round-robin and store their states;
// a second phase merges every (row, head) over its spans.
//
// Cross-workgroup data is written with write-through (agent-scope) stores
// and every activation buffer is written once per launch (per-layer
// buffers), so no workgroup can read a stale line from its XCD's L2.
// Every wait is bounded: on timeout the kernel raises an error flag and all
// waves still run to the end.
//
// Tiles are the same units with the same arithmetic as the per-operation
// kernels (tiles.h), so results match those kernels bit for bit.
#include "attn.h"

namespace as2d {

// Phase counter layout (phase_cnt): 0 embedded rows; per layer l, base
// 1 + 6 l: +0 QKV, +1 attention chunk tiles, +2 merged (row, head) pairs,
// +3 O, +4 gate/up, +5 down; then the LM head (1 + 6 L) and verified rows
// (2 + 6 L).  A GEMM phase counts the signals of its G workgroups.
__device__ __forceinline__ int ph_layer(int l, int k) { return 1 + 6 * l + k; }

__device__ __forceinline__ void signal_done(int* c) {
  __syncthreads();  // waits for every wave's stores, then joins
  if (threadIdx.x == 0) counter_add(c, 1);
}

// Waits until *c >= target.  Bounded: after spin_limit polls the error
// flag is raised; once it is raised (by any workgroup) every wait returns
// at once, so all waves reach the end of the kernel.
__device__ __forceinline__ void wait_count(const int* c, int target, int* err, int spin_limit) {
  if (threadIdx.x == 0) {
    int n = 0;
    for (;;) {
      const int v = ld_coherent(c), e = ld_coherent(err);   // one round trip per poll
      if (v >= target || e) break;
      __builtin_amdgcn_s_sleep(1);
      if (++n > spin_limit) {
        st<true>(err, 1);
        break;
      }
    }
  }
  lds_sync();  // the weight prefetch stays in flight
}

// Optional timeline: stamps (phase entry, inputs ready, phase exit) of each
// workgroup, in wall-clock ticks.
__device__ __forceinline__ void stamp(const StepArgs& a, int phase, int which) {
  if (a.trace && threadIdx.x == 0)
    a.trace[((size_t)blockIdx.x * (3 + 6 * a.n_layers) + phase) * 3 + which] = wall_clock64();
}

// One GEMM phase of a balanced plan: workgroup b < G streams its share of
// the (pair, split) units (the same units and sums as the balanced
// kernel), issuing its first weight loads before the wait for the
// producer, and signals once its partials, fixups and epilogues are
// stored, so the phase is done at G signals.
template <bool BF, int MT, int SL, int AM, int EPI>
__device__ __forceinline__ void gemm_phase(const GemmArgs& p, int M, const int* wait_c, int wait_target, int* done_c,
                           const StepArgs& a, unsigned char* smem, float* s_scale, int* s_flags) {
  const int phase = (int)(done_c - a.phase_cnt);
  stamp(a, phase, 0);
  bool waited = false;
  auto wait = [&] {
    if (!waited) {
      wait_count(wait_c, wait_target, a.err, a.spin_limit);
      stamp(a, phase, 1);
      waited = true;
    }
  };
  if ((int)blockIdx.x < p.G) {
    bool ra = false;
    if constexpr (SL > 0 && MT == 1 && AM == A_NORM && (EPI == EPI_SWIGLU || EPI == EPI_ARGMAX)) {
      if (range_ra_slice<BF>(AM, EPI, MT, p.KS, p.KT) == SL) {
        constexpr int P = SL % kRangePrefetch == 0 ? kRangePrefetch : SL;
        gemm_range_direct_ra<BF, P, SL, AM, EPI, true>(p, M, smem, s_scale, s_flags, wait);
        ra = true;
      }
    }
    if (!ra) gemm_range_direct<BF, MT, kRangePrefetch, AM, EPI, true>(p, M, smem, s_scale, s_flags, wait);
    wait_vmem();
    signal_done(done_c);
  }
  stamp(a, phase, 2);
}

// SL: slice length of the register-resident balanced variant for the
// gate/up and LM-head phases (0: none).  One workgroup per compute unit.
template <bool BF, int MT, int D, int SL>
__global__ __launch_bounds__(256, 1) void step_kernel(const StepArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ float s_scale[kMaxRows];
  __shared__ int s_flags[kMaxUnits];
  __shared__ int s_tok, s_bad;
  __shared__ float s_margin;
  __shared__ float s4f[4], s4s[4];
  __shared__ int s4i[4];
  const int G = gridDim.x, tid = threadIdx.x;
  const int M = a.M, L = a.n_layers;

  // embedding rows
  stamp(a, 0, 0);
  for (int m = blockIdx.x; m < M; m += G) {
    embed_row<BF, true>(a.rows, m, (const typename ET<BF>::T*)a.embed, (const typename ET<BF>::T*)a.audio,
                        a.hidden, a.gain0, a.x0, a.sumsq0, a.xg0, a.xg0_plane, reinterpret_cast<float*>(smem));
    signal_done(&a.phase_cnt[0]);
  }

  stamp(a, 0, 2);
  // attention items of this pass: (request, 128-key span, query head)
  // attention items: (request, span, KV head, 16-row block of the rows of
  // the query heads that share the KV head), as in the per-operation kernel
  const int hpg = a.n_q / a.n_kv;
  int n_items = 0;
  for (int r = 0; r < a.n_reqs; ++r) {
    const ReqDesc rq = load_invariant(a.reqs + r);
    n_items += a.n_kv * ((hpg * rq.W + 15) / 16) * ((rq.L0 + rq.W - 1) / kAttnSpanKeys + 1);
  }
  constexpr int KS = D / AttnFmt<BF>::KE;
  const int quarter = tid >> 4;

  for (int l = 0; l < L; ++l) {
    const StepLayer* ly = a.layers + l;
    const int* prev = l == 0 ? &a.phase_cnt[0] : &a.phase_cnt[ph_layer(l - 1, 5)];
    const int prev_target = l == 0 ? M : a.done_down;
    gemm_phase<BF, MT, SL, A_NORM, EPI_QKV>(load_invariant(&ly->qkv), M, prev, prev_target, &a.phase_cnt[ph_layer(l, 0)], a, smem,
                                             s_scale, s_flags);

    // attention spans, dealt round-robin; each item stores its rows' span
    // states
    stamp(a, ph_layer(l, 1), 0);
    if ((int)blockIdx.x < n_items) {
      wait_count(&a.phase_cnt[ph_layer(l, 0)], a.done_qkv, a.err, a.spin_limit);
      stamp(a, ph_layer(l, 1), 1);
      const AttnArgs at = load_invariant(&ly->attn);
      int mine = 0;
      for (int t = blockIdx.x; t < n_items; t += G) {
        int r = 0, u = t, ns = 0, nb = 0;
        ReqDesc rq;
        for (;; ++r) {
          rq = load_invariant(a.reqs + r);
          ns = (rq.L0 + rq.W - 1) / kAttnSpanKeys + 1;
          nb = (hpg * rq.W + 15) / 16;
          if (u < a.n_kv * nb * ns || r == a.n_reqs - 1) break;
          u -= a.n_kv * nb * ns;
        }
        const int sp = u / (a.n_kv * nb);
        const int v = u - sp * a.n_kv * nb;
        const int g = v / nb, b = v - g * nb;
        const AttnRows rows{g * hpg, rq.W, hpg * rq.W, 16 * b};
        Op2 q[1][KS];
        attn_load_q<BF, D, 1>(at, rq, rows, q);
        AttnState<1, D / 64> sst;
        attn_span<BF, D, 1>(at, rq, rows, sp, q, smem, sst);
        attn_store_span<D, 1>(at, rq, rows, sp, sst);
        lds_sync();   // the next item writes the LDS again
        ++mine;
      }
      // one signal for all this workgroup's items, once their stores are done
      wait_vmem();
      __syncthreads();
      if (tid == 0) counter_add(&a.phase_cnt[ph_layer(l, 1)], mine);
    }
    stamp(a, ph_layer(l, 1), 2);

    // merge of every (row, head), one per quarter wave, spans in ascending order
    const int n_merge = M * a.n_q;
    stamp(a, ph_layer(l, 2), 0);
    if ((int)blockIdx.x * 16 < n_merge) {
      wait_count(&a.phase_cnt[ph_layer(l, 1)], n_items, a.err, a.spin_limit);
      stamp(a, ph_layer(l, 2), 1);
      const AttnArgs at = load_invariant(&ly->attn);
      int mine = 0;
      for (int t0 = blockIdx.x * 16; t0 < n_merge; t0 += G * 16) {
        const int t = t0 + quarter;
        if (t < n_merge) {
          const int m = t / a.n_q, h = t - m * a.n_q;
          int r = 0;
          ReqDesc rq = load_invariant(a.reqs);
          while (r < a.n_reqs - 1 && m >= rq.row_start + rq.W) rq = load_invariant(a.reqs + ++r);
          attn_merge_row<BF, D, true>(at, rq, m - rq.row_start, h);
        }
        mine += min(16, n_merge - t0);
      }
      wait_vmem();
      __syncthreads();
      if (tid == 0) counter_add(&a.phase_cnt[ph_layer(l, 2)], mine);
    }
    stamp(a, ph_layer(l, 2), 2);

    gemm_phase<BF, MT, SL, A_PLAIN, EPI_RESID>(load_invariant(&ly->o), M, &a.phase_cnt[ph_layer(l, 2)], n_merge,
                                                &a.phase_cnt[ph_layer(l, 3)], a, smem, s_scale, s_flags);
    gemm_phase<BF, MT, SL, A_NORM, EPI_SWIGLU>(load_invariant(&ly->gu), M, &a.phase_cnt[ph_layer(l, 3)], a.done_o,
                                                &a.phase_cnt[ph_layer(l, 4)], a, smem, s_scale, s_flags);
    gemm_phase<BF, MT, SL, A_PLAIN, EPI_DOWN>(load_invariant(&ly->down), M, &a.phase_cnt[ph_layer(l, 4)], a.done_gu,
                                                &a.phase_cnt[ph_layer(l, 5)], a, smem, s_scale, s_flags);
  }
  gemm_phase<BF, MT, SL, A_NORM, EPI_ARGMAX>(a.lm, M, &a.phase_cnt[ph_layer(L - 1, 5)], a.done_down,
                                              &a.phase_cnt[1 + 6 * L], a, smem, s_scale, s_flags);

  // arg-max of each verified row on the last workgroups, then verification
  // by the last row to finish
  for (int i = G - 1 - blockIdx.x; i < a.fin_rows; i += G) {
    int r = 0, u = i;
    while (r < a.n_fin - 1 && u >= load_invariant(a.fin_reqs + r).W) u -= load_invariant(a.fin_reqs + r++).W;
    const int row = load_invariant(a.fin_reqs + r).row_start + u;
    wait_count(&a.phase_cnt[1 + 6 * L], a.done_lm, a.err, a.spin_limit);
    argmax_row<true>(a.lm.amax_val, a.lm.amax_val2, a.lm.amax_idx, a.lm.N / kPairCols, row, &s_tok, &s_bad,
                     &s_margin, s4f, s4s, s4i);
    if (tid == 0) {
      st<true>(a.row_tok + row, s_tok);
      st<true>(a.row_bad + row, s_bad);
      a.row_margin[row] = s_margin;   // read by the host after the pass
      wait_vmem();
      if (counter_add(&a.phase_cnt[2 + 6 * L], 1) == a.fin_rows - 1) {
        for (int q = 0; q < a.n_fin; ++q) {
          const ReqDesc rq = load_invariant(a.fin_reqs + q);
          int bad = 0;
          for (int w = 0; w < rq.W; ++w) bad |= ld_coherent(a.row_bad + rq.row_start + w);
          a.out[q] = verify_request(a.rows, rq, [&](int rr) { return ld_coherent(a.row_tok + rr); }, bad);
        }
      }
    }
    __syncthreads();
  }
}

// Clears the phase counters before a launch (a kernel rather than a memset
// so that the pair can be captured into a graph).
__global__ void clear_kernel(int* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

template <bool BF, int MT, int D, int SL>
static const void* step_fn() {
  return reinterpret_cast<const void*>(&step_kernel<BF, MT, D, SL>);
}

// The instantiated kernels: (bf16, MT, head_dim, SL) for SL = 0 and the
// register-resident slice lengths (one row tile only).
template <bool BF, int D>
static const void* pick_sl(int MT, int SL) {
  if (MT == 2) return step_fn<BF, 2, D, 0>();
  if (SL == kRangeSL<BF>[0]) return step_fn<BF, 1, D, kRangeSL<BF>[0]>();
  if (SL == kRangeSL<BF>[1]) return step_fn<BF, 1, D, kRangeSL<BF>[1]>();
  if (SL == kRangeSL<BF>[2]) return step_fn<BF, 1, D, kRangeSL<BF>[2]>();
  return step_fn<BF, 1, D, 0>();
}

static const void* pick(bool bf16, int MT, int D, int SL) {
  if (D == 128) return bf16 ? pick_sl<true, 128>(MT, SL) : pick_sl<false, 128>(MT, SL);
  return bf16 ? pick_sl<true, 64>(MT, SL) : pick_sl<false, 64>(MT, SL);
}

int step_ra_slice(bool bf16, int KS, int KT) {
  return bf16 ? range_ra_slice<true>(A_NORM, EPI_SWIGLU, 1, KS, KT)
              : range_ra_slice<false>(A_NORM, EPI_SWIGLU, 1, KS, KT);
}

int step_lds_bytes(int MT, int head_dim, int hidden) {
  // hidden <= 8192
  int b = kRangeMinLds;                                 // one workgroup per compute unit
  b = max(b, gemm_range_lds_bytes(MT, kMaxUnits));
  b = max(b, head_dim == 128 ? attn_span_lds_bytes<true, 128, 2>() : attn_span_lds_bytes<true, 64, 2>());
  b = max(b, head_dim == 128 ? attn_span_lds_bytes<false, 128, 2>() : attn_span_lds_bytes<false, 64, 2>());
  b = max(b, hidden * 4);                               // embedding row
  return b;
}

hipError_t prepare_step_kernels() {
  for (int bf = 0; bf < 2; ++bf)
    for (int d = 64; d <= 128; d += 64)
      for (int mt = 1; mt <= 2; ++mt)
        for (int i = -1; i < 3; ++i) {
          const int sl = i < 0 ? 0 : (bf ? kRangeSL<true>[i] : kRangeSL<false>[i]);
          hipError_t e = hipFuncSetAttribute(pick(bf, mt, d, sl), hipFuncAttributeMaxDynamicSharedMemorySize,
                                             step_lds_bytes(mt, d, 8192));
          if (e != hipSuccess) return e;
        }
  return hipSuccess;
}

hipError_t step_occupancy(bool bf16, int MT, int head_dim, int hidden, int sl, int* blocks_per_cu) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, pick(bf16, MT, head_dim, sl), 256,
                                                      step_lds_bytes(MT, head_dim, hidden));
}

hipError_t launch_step(bool bf16, int MT, int head_dim, int sl, const StepArgs& a, int grid, int n_counters,
                       hipStream_t s) {
  clear_kernel<<<8, 256, 0, s>>>(a.phase_cnt, n_counters);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const void* fn = pick(bf16, MT, head_dim, sl);
  void* args[] = {const_cast<StepArgs*>(&a)};
  return hipLaunchKernel(fn, dim3(grid), dim3(256), args, step_lds_bytes(MT, head_dim, a.hidden), s);
}

}  // namespace as2d
