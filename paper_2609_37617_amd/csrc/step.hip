// Persistent step kernel: one launch runs a whole verification pass
// (embedding, every decoder layer, LM head and greedy verification) for up
// to 32 rows.
//
// All workgroups are resident at once (grid = occupancy x CUs).  The pass
// is a sequence of phases; a phase's tiles are dealt round-robin to the
// workgroups, which walk the phases in order.  A tile that consumes the
// previous phase's output first issues its weight loads (weights do not
// depend on activations), then waits until the producing phase's
// completion counter reaches its target, so weight streaming continues
// across phase boundaries instead of stopping at a kernel boundary.
//
// Cross-workgroup data is written with write-through (agent-scope) stores
// and every activation buffer is written once per launch (per-layer
// buffers), so no workgroup can read a stale line from its XCD's L2.
// Every wait is bounded: on timeout the kernel raises an error flag and all
// waves still run to the end.
//
// Tiles are the same units with the same arithmetic as the per-operation
// kernels (tiles.h), so results match those kernels bit for bit.
#include "tiles.h"

namespace as2d {

// Phase counter layout (phase_cnt): 0 embedding; per layer l, base 1 + 6 l:
// +0 QKV tile pairs, +1 attention chunk tiles, +2 merged (row, head) pairs,
// +3 O tile pairs, +4 gate/up tile pairs, +5 down tile pairs; then LM head
// tile pairs (1 + 6 L) and verified rows (2 + 6 L).
__device__ __forceinline__ int ph_layer(int l, int k) { return 1 + 6 * l + k; }

__device__ __forceinline__ void signal_done(int* c) {
  __syncthreads();  // waits for every wave's stores, then joins
  if (threadIdx.x == 0) counter_add(c, 1);
}

// Waits until *c >= target.  Bounded: after spin_limit polls the error
// flag is raised; once it is raised (by any workgroup) every wait returns
// at once, so all waves reach the end of the kernel.
__device__ __noinline__ void wait_count(const int* c, int target, int* err, int spin_limit) {
  if (threadIdx.x == 0) {
    int n = 0;
    while (ld_coherent(c) < target) {
      if (ld_coherent(err)) break;
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

template <bool BF, int MT, int AM, int EPI>
__device__ void gemm_phase(const GemmArgs p, int M, const int* wait_c, int wait_target, int* done_c,
                           const StepArgs& a, unsigned char* smem, float* s_scale, int* s_flag) {
  const int G = gridDim.x;
  const int n_tiles = (p.N / kPairCols) * p.KS;
  const int phase = (int)(done_c - a.phase_cnt);
  stamp(a, phase, 0);
  bool waited = false;
  for (int t = blockIdx.x; t < n_tiles; t += G) {
    const int pair = t / p.KS, split = t - pair * p.KS;
    const bool fin = gemm_tile_direct<BF, MT, 1, kWaves, false, AM, EPI, true, true>(p, M, pair, split, smem, s_scale, s_flag, [&] {
      if (!waited) {
        wait_count(wait_c, wait_target, a.err, a.spin_limit);
        stamp(a, phase, 1);
        waited = true;
      }
    });
    if (fin) signal_done(done_c);
  }
  stamp(a, phase, 2);
}

template <bool BF, int MT, int D>
__global__ __launch_bounds__(256, 2) void step_kernel(const StepArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ float s_scale[kMaxRows];
  __shared__ int s_flag, s_tok, s_bad;
  __shared__ float s4f[4];
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
  // attention tiles of this pass: n_q heads x chunks of each request
  int n_chunk_tiles = 0;
  for (int r = 0; r < a.n_reqs; ++r)
    n_chunk_tiles += a.n_q * ((a.reqs[r].L0 + a.reqs[r].W + kAttnChunk - 1) / kAttnChunk);
  constexpr int kMergeGroups = 256 / D;  // (row, head) merges per workgroup pass

  for (int l = 0; l < L; ++l) {
    const StepLayer& ly = a.layers[l];
    const int* prev = l == 0 ? &a.phase_cnt[0] : &a.phase_cnt[ph_layer(l - 1, 5)];
    const int prev_target = l == 0 ? M : a.pairs_down;
    gemm_phase<BF, MT, A_NORM, EPI_QKV>(ly.qkv, M, prev, prev_target, &a.phase_cnt[ph_layer(l, 0)], a, smem,
                                         s_scale, &s_flag);

    // attention chunks
    stamp(a, ph_layer(l, 1), 0);
    bool waited = false;
    for (int t = blockIdx.x; t < n_chunk_tiles; t += G) {
      int r = 0, u = t;
      for (;; ++r) {
        const int n = a.n_q * ((a.reqs[r].L0 + a.reqs[r].W + kAttnChunk - 1) / kAttnChunk);
        if (u < n || r == a.n_reqs - 1) break;
        u -= n;
      }
      const ReqDesc rq = a.reqs[r];
      const int nch = (rq.L0 + rq.W + kAttnChunk - 1) / kAttnChunk;
      const int h = u / nch, c = u - h * nch;
      if (!waited) {
        wait_count(&a.phase_cnt[ph_layer(l, 0)], a.pairs_qkv, a.err, a.spin_limit);
        stamp(a, ph_layer(l, 1), 1);
        waited = true;
      }
      const AttnArgs at = ly.attn;
      attn_chunk_tile<D, true>(at, c, h, rq, smem);
      signal_done(&a.phase_cnt[ph_layer(l, 1)]);
    }
    stamp(a, ph_layer(l, 1), 2);

    // merge of every (row, head): kMergeGroups per workgroup pass
    const int n_merge = M * a.n_q;
    stamp(a, ph_layer(l, 2), 0);
    waited = false;
    for (int t0 = blockIdx.x * kMergeGroups; t0 < n_merge; t0 += G * kMergeGroups) {
      if (!waited) {
        wait_count(&a.phase_cnt[ph_layer(l, 1)], n_chunk_tiles, a.err, a.spin_limit);
        stamp(a, ph_layer(l, 2), 1);
        waited = true;
      }
      const int grp = tid / D;
      const int t = t0 + grp;
      float* sm = reinterpret_cast<float*>(smem) + grp * 2 * kMaxChunks;
      const AttnArgs at = ly.attn;
      if (t < n_merge)
        attn_merge_row<BF, D, true>(at, t / a.n_q, t % a.n_q, grp * D, sm, sm + kMaxChunks,
                                    [] { __syncthreads(); }, true);
      else
        attn_merge_row<BF, D, true>(at, 0, 0, grp * D, sm, sm + kMaxChunks, [] { __syncthreads(); },
                                    false);
      __syncthreads();
      if (tid == 0) counter_add(&a.phase_cnt[ph_layer(l, 2)], min(kMergeGroups, n_merge - t0));
    }
    stamp(a, ph_layer(l, 2), 2);

    gemm_phase<BF, MT, A_PLAIN, EPI_RESID>(ly.o, M, &a.phase_cnt[ph_layer(l, 2)], n_merge,
                                            &a.phase_cnt[ph_layer(l, 3)], a, smem, s_scale, &s_flag);
    gemm_phase<BF, MT, A_NORM, EPI_SWIGLU>(ly.gu, M, &a.phase_cnt[ph_layer(l, 3)], a.pairs_o,
                                            &a.phase_cnt[ph_layer(l, 4)], a, smem, s_scale, &s_flag);
    gemm_phase<BF, MT, A_PLAIN, EPI_RESID>(ly.down, M, &a.phase_cnt[ph_layer(l, 4)], a.pairs_gu,
                                            &a.phase_cnt[ph_layer(l, 5)], a, smem, s_scale, &s_flag);
  }
  gemm_phase<BF, MT, A_NORM, EPI_ARGMAX>(a.lm, M, &a.phase_cnt[ph_layer(L - 1, 5)], a.pairs_down,
                                          &a.phase_cnt[1 + 6 * L], a, smem, s_scale, &s_flag);

  // arg-max of each verified row on the last workgroups, then verification
  // by the last row to finish
  for (int i = G - 1 - blockIdx.x; i < a.fin_rows; i += G) {
    int r = 0, u = i;
    while (r < a.n_fin - 1 && u >= a.fin_reqs[r].W) u -= a.fin_reqs[r++].W;
    const int row = a.fin_reqs[r].row_start + u;
    wait_count(&a.phase_cnt[1 + 6 * L], a.pairs_lm, a.err, a.spin_limit);
    argmax_row<true>(a.lm.amax_val, a.lm.amax_idx, a.lm.N / kPairCols, row, &s_tok, &s_bad, s4f, s4i);
    if (tid == 0) {
      st<true>(a.row_tok + row, s_tok);
      st<true>(a.row_bad + row, s_bad);
      wait_vmem();
      if (counter_add(&a.phase_cnt[2 + 6 * L], 1) == a.fin_rows - 1) {
        for (int q = 0; q < a.n_fin; ++q) {
          const ReqDesc rq = a.fin_reqs[q];
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

template <bool BF, int MT, int D>
static const void* step_fn() {
  return reinterpret_cast<const void*>(&step_kernel<BF, MT, D>);
}

static const void* pick(bool bf16, int MT, int D) {
  if (D == 128) {
    if (bf16) return MT == 1 ? step_fn<true, 1, 128>() : step_fn<true, 2, 128>();
    return MT == 1 ? step_fn<false, 1, 128>() : step_fn<false, 2, 128>();
  }
  if (bf16) return MT == 1 ? step_fn<true, 1, 64>() : step_fn<true, 2, 64>();
  return MT == 1 ? step_fn<false, 1, 64>() : step_fn<false, 2, 64>();
}

int step_lds_bytes(int head_dim, int hidden) {
  // hidden <= 8192
  int b = gemm_direct_lds_bytes<2, 1>(kMaxSlices);
  b = max(b, head_dim == 128 ? attn_lds_bytes<128>() : attn_lds_bytes<64>());
  b = max(b, hidden * 4);                      // embedding row
  b = max(b, (256 / head_dim) * 2 * kMaxChunks * 4);  // merge scratch
  return b;
}

hipError_t prepare_step_kernels() {
  const int lds128 = step_lds_bytes(128, 8192), lds64 = step_lds_bytes(64, 8192);
  const void* fns[8] = {step_fn<true, 1, 128>(), step_fn<true, 2, 128>(), step_fn<false, 1, 128>(),
                        step_fn<false, 2, 128>(), step_fn<true, 1, 64>(),  step_fn<true, 2, 64>(),
                        step_fn<false, 1, 64>(),  step_fn<false, 2, 64>()};
  for (int i = 0; i < 8; ++i) {
    hipError_t e = hipFuncSetAttribute(fns[i], hipFuncAttributeMaxDynamicSharedMemorySize, i < 4 ? lds128 : lds64);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t step_occupancy(bool bf16, int MT, int head_dim, int hidden, int* blocks_per_cu) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks_per_cu, pick(bf16, MT, head_dim), 256,
                                                      step_lds_bytes(head_dim, hidden));
}

hipError_t launch_step(bool bf16, int MT, int head_dim, const StepArgs& a, int grid, int n_counters,
                       hipStream_t s) {
  clear_kernel<<<8, 256, 0, s>>>(a.phase_cnt, n_counters);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = step_lds_bytes(head_dim, a.hidden);
#define AS2D_S(bf, mt, d) step_kernel<bf, mt, d><<<grid, 256, lds, s>>>(a)
  if (head_dim == 128) {
    if (bf16) { if (MT == 1) AS2D_S(true, 1, 128); else AS2D_S(true, 2, 128); }
    else { if (MT == 1) AS2D_S(false, 1, 128); else AS2D_S(false, 2, 128); }
  } else {
    if (bf16) { if (MT == 1) AS2D_S(true, 1, 64); else AS2D_S(true, 2, 64); }
    else { if (MT == 1) AS2D_S(false, 1, 64); else AS2D_S(false, 2, 64); }
  }
#undef AS2D_S
  return hipGetLastError();
}

}  // namespace as2d
