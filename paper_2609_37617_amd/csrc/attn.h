// Block-causal grouped-query attention of the verification step on matrix
// cores, shared by the per-operation kernels (kernels.hip) and the
// persistent step kernel (step.hip).
//
// Arithmetic of one row (position pos) and query head h, reading KV head
// g = floor(h n_kv / n_q).  Keys are taken in blocks of kAttnBlock = 64 at
// absolute positions; block b holds keys [64 b, 64 b + 64) up to pos:
//   s_j   = (q . k_j) * scale, a matrix-core product: for bf16 models q and
//           k are split into bf16 pairs (hi = bf16(x), lo = bf16(x - hi))
//           and s = q_hi k_hi + q_hi k_lo + q_lo k_hi over four 32-wide
//           k-steps; float32 models use float32 products;
//   m_b   = max_j s_j (per 16-key tile, then the four tiles);
//   p_j   = exp(s_j - m_b), 0 for keys after pos;
//   l_b   = sum_j p_j: per 16-key tile in a fixed butterfly, the four tile
//           sums added in order;
//   acc_b = sum_j p_j v_j, a matrix-core product of the (hi, lo) splits of
//           p and v (p_hi v_hi + p_hi v_lo + p_lo v_hi, 32-key steps).
// s is formed transposed (keys on the matrix-core rows), so each lane holds
// four consecutive keys of one query row; the sums over keys run in a fixed
// pattern (a lane's four keys in order, then across lanes in a fixed
// butterfly, then the four 16-key tiles in order).
// Merging a partial (m, l, acc) into a running state (M, L, A):
//   M' = max(M, m), a = exp(M - M'), c = exp(m - M'),
//   L = fma(L, a, l c), A = fma(A, a, acc c), M = M'.
// Two levels: the blocks of each span of kAttnSpan = 2 blocks (128 keys,
// absolute) are merged in ascending order, starting from the span's first
// block; the spans' states are then merged in ascending order, starting
// from span 0.  The output is A / L.
//
// Every quantity of a row depends only on that row's query and the keys
// and values (matrix-core rows are independent), so a row gets the same
// bits whatever other rows share its tile and whoever merges its spans:
// the verification kernel (spans on different workgroups, span states
// through memory) or the prefill kernel (spans in a loop, in registers).
#pragma once
#include "tiles.h"

namespace as2d {

template <bool BF> struct AttnFmt {
  static constexpr int PER = BF ? 8 : 4;                  // elements per lane per k-step
  static constexpr int KE = 4 * PER;                      // k-step
  static constexpr int PARTS = BF ? 2 : 1;                // hi, lo planes
  static constexpr int VS = kAttnBlock + (BF ? 8 : 4);    // LDS row stride of V^T and P, elements
  static constexpr int ES = BF ? 2 : 4;                   // bytes per LDS element
};

// LDS of a block tile for RT row tiles: P [PARTS][16 RT][VS] and the
// per-wave row statistics [2][4][16 RT] floats.
template <bool BF, int D, int RT> __host__ __device__ constexpr int attn_block_lds_bytes() {
  using F = AttnFmt<BF>;
  return F::PARTS * 16 * RT * F::VS * F::ES + 2 * 4 * 16 * RT * 4;
}

// A matrix-core operand of one k-step (16 bytes per lane and part).
struct Op2 {
  uint4 h, l;
};

// (hi, lo) split of PER consecutive floats (bf16: 8 floats into two sets
// of eight bf16; float32: 4 floats as they are).
template <bool BF> __device__ __forceinline__ Op2 split_op(const float4* v) {
  Op2 o;
  if constexpr (BF) {
    const float e[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint16_t h0 = f2bf(e[2 * t]), h1 = f2bf(e[2 * t + 1]);
      const uint16_t l0 = f2bf(e[2 * t] - bf2f(h0)), l1 = f2bf(e[2 * t + 1] - bf2f(h1));
      hw[t] = h0 | ((uint32_t)h1 << 16);
      lw[t] = l0 | ((uint32_t)l1 << 16);
    }
    o.h = make_uint4(hw[0], hw[1], hw[2], hw[3]);
    o.l = make_uint4(lw[0], lw[1], lw[2], lw[3]);
  } else {
    o.h = make_uint4(__float_as_uint(v[0].x), __float_as_uint(v[0].y), __float_as_uint(v[0].z),
                     __float_as_uint(v[0].w));
    o.l = o.h;
  }
  return o;
}

// q_hi k_hi + q_hi k_lo + q_lo k_hi (bf16) or the float32 product, in that order.
template <bool BF> __device__ __forceinline__ f4 mma3(const Op2& a, const Op2& b, f4 acc) {
  if constexpr (BF) {
    acc = mma_step<true>(a.h, b.h, acc);
    acc = mma_step<true>(a.h, b.l, acc);
    acc = mma_step<true>(a.l, b.h, acc);
  } else {
    acc = mma_step<false>(a.h, b.h, acc);
  }
  return acc;
}

// Reduction over the 16 lanes of a DPP row (the lanes that hold the same
// four rows of a matrix-core tile): each step combines the same two values
// on both partner lanes, so all 16 lanes end with the same bits.
template <class Op> __device__ __forceinline__ float row16_reduce(float v, Op op) {
  v = op(v, dpp_get<kDppXor1>(v));
  v = op(v, dpp_get<kDppXor2>(v));
  v = op(v, dpp_get<kDppHalfMirror>(v));
  return op(v, dpp_get<kDppMirror>(v));
}

// Combination with the partner lane l ^ 16 (SWAP32 false) or l ^ 32 (true)
// through the cross-row swaps of gfx950: both partners receive the pair
// (lower lane's value, upper lane's value) in that order and so end with the
// same bits.
template <bool SWAP32, class Op> __device__ __forceinline__ float swap_combine(float v, Op op) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v);
  uint32_t lo, hi;
  if constexpr (SWAP32) {
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    lo = r[0];
    hi = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    lo = r[0];
    hi = r[1];
  }
  return op(__builtin_bit_cast(float, lo), __builtin_bit_cast(float, hi));
}
struct FMax {
  __device__ float operator()(float a, float b) const { return fmaxf(a, b); }
};
struct FAdd {
  __device__ float operator()(float a, float b) const { return a + b; }
};

// Merge of a partial (m, l) into the running (M, L): the coefficients of
// the running and the new sums.
struct MergeCoef {
  float a, c;
};
__device__ __forceinline__ MergeCoef attn_merge_coef(float& M, float& L, float m, float l) {
#pragma clang fp contract(off)
  const float Mn = fmaxf(M, m);
  const MergeCoef k{expf(M - Mn), expf(m - Mn)};
  L = __builtin_fmaf(L, k.a, l * k.c);
  M = Mn;
  return k;
}
__device__ __forceinline__ float attn_merge_acc(float A, float acc, MergeCoef k) {
#pragma clang fp contract(off)
  return __builtin_fmaf(A, k.a, acc * k.c);
}

// The operands of one request's queries for head h: this lane's share of
// every k-step of row tiles rt < RT (rows 16 rt + lane % 16 of the request;
// rows past W read row W - 1, whose results are never used).
template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_load_q(const AttnArgs& p, const ReqDesc& rq, int h, Op2 (&q)[RT][D / AttnFmt<BF>::KE]) {
  using F = AttnFmt<BF>;
  const int lane = threadIdx.x & 63;
  const int qcols = p.n_q * D;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = min(16 * rt + (lane & 15), rq.W - 1);
    const float4* base =
        reinterpret_cast<const float4*>(p.q + (size_t)(rq.row_start + r) * qcols + h * D + F::PER * (lane >> 4));
#pragma unroll
    for (int ks = 0; ks < D / F::KE; ++ks) {
      float4 v[2];
      v[0] = ldg(base + F::KE / 4 * ks);
      if constexpr (BF) v[1] = ldg(base + F::KE / 4 * ks + 1);
      q[rt][ks] = split_op<BF>(v);
    }
  }
}

// One block's keys and values as loaded from the cache (layout: AttnArgs),
// already the matrix-core operands: lane l of wave w holds the k-step
// slices of key 16 w + l % 16 (for s, rows of the transposed product) and,
// for each of its dimension tiles t, dimension 16 (w DTW + t) + l % 16 at
// keys KE ks + PER (l / 16) + e (for p v).  Keys past the request's: K
// reads its last key (a branch-free load, never used), V elements are set
// to zero (their p is 0, and 0 times a stale value must stay 0).
template <bool BF, int D> struct AttnRaw {
  static constexpr int KS = D / AttnFmt<BF>::KE;
  static constexpr int KSV = kAttnBlock / AttnFmt<BF>::KE;
  static constexpr int DTW = D / 64;
  Op2 k[KS];
  Op2 v[DTW][KSV];
};

// Zeroes the elements e of a 16-byte operand (bf16: 8, float32: 4) whose
// index is at least n (n in [0, PER]).
template <bool BF> __device__ __forceinline__ uint4 keep_first(uint4 x, int n) {
  uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if constexpr (BF) {
      const uint32_t lo = 2 * t < n ? 0x0000ffffu : 0u, hi = 2 * t + 1 < n ? 0xffff0000u : 0u;
      w[t] &= lo | hi;
    } else {
      w[t] = t < n ? w[t] : 0u;
    }
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <bool BF, int D>
__device__ __forceinline__ void attn_fetch(const AttnArgs& p, const ReqDesc& rq, int h, int b, AttnRaw<BF, D>& r) {
  using F = AttnFmt<BF>;
  using Raw = AttnRaw<BF, D>;
  using T = typename ET<BF>::T;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lg = lane >> 4, lr = lane & 15;
  const int key0 = b * kAttnBlock;
  const int last = rq.L0 + rq.W - 1;          // last key of the request in this pass
  const int g = h * p.n_kv / p.n_q;
  const size_t head = (size_t)rq.slot * p.slot_stride + (size_t)g * p.kv_cap * D;   // float32 units
  const T* kb = reinterpret_cast<const T*>(p.k_cache + head);
  const T* vb = reinterpret_cast<const T*>(p.v_cache + head);
  const T* kr = kb + (size_t)min(key0 + 16 * wave + lr, last) * F::PARTS * D + F::PER * lg;
#pragma unroll
  for (int ks = 0; ks < Raw::KS; ++ks) {
    r.k[ks].h = ldg(reinterpret_cast<const uint4*>(kr + F::KE * ks));
    r.k[ks].l = BF ? ldg(reinterpret_cast<const uint4*>(kr + D + F::KE * ks)) : r.k[ks].h;
  }
  const bool tail = key0 + kAttnBlock > last + 1;   // the block holds keys past the request's
#pragma unroll
  for (int t = 0; t < Raw::DTW; ++t) {
    const T* vr = vb + (size_t)(16 * (wave * Raw::DTW + t) + lr) * p.kv_cap + key0 + F::PER * lg;
#pragma unroll
    for (int ks = 0; ks < Raw::KSV; ++ks) {
      Op2 o;
      o.h = ldg(reinterpret_cast<const uint4*>(vr + F::KE * ks));
      o.l = BF ? ldg(reinterpret_cast<const uint4*>(vr + (size_t)D * p.kv_cap + F::KE * ks)) : o.h;
      if (tail) {
        const int n = min(max(last + 1 - (key0 + F::KE * ks + F::PER * lg), 0), F::PER);
        o.h = keep_first<BF>(o.h, n);
        o.l = keep_first<BF>(o.l, n);
      }
      r.v[t][ks] = o;
    }
  }
}

// One block of keys (block b) of request rq, rows of row tiles rt < RT
// (queries q; keys and values of the query head's KV head as fetched in
// raw): the block statistics of every row and acc_b of this wave's
// dimension tiles.  256 threads, 4 waves: wave w forms s for keys
// [16 w, 16 w + 16) of the block and acc_b for dimension tiles
// [w DTW, (w + 1) DTW).  On return, for lane l and i < 4, row
// 16 rt + 4 (l / 16) + i has statistics m[rt][i], l[rt][i] (m = -inf, l = 0
// when the block starts after the row's position) and acc[rt][t] holds
// acc_b of that row at dimension 16 (w DTW + t) + l % 16.  smem:
// attn_block_lds_bytes<BF, D, RT>(), not in use on entry (the caller
// synchronises the workgroup between blocks).
template <bool BF, int D, int RT> struct AttnBlockOut {
  static constexpr int DTW = D / 64;   // dimension tiles per wave
  f4 acc[RT][DTW];
  float m[RT][4], l[RT][4];
};

template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_block(const AttnArgs& p, const ReqDesc& rq, int b,
                                           const Op2 (&q)[RT][D / AttnFmt<BF>::KE], const AttnRaw<BF, D>& raw,
                                           unsigned char* smem, AttnBlockOut<BF, D, RT>& out) {
#pragma clang fp contract(off)
  using F = AttnFmt<BF>;
  using T = typename ET<BF>::T;
  constexpr int KS = D / F::KE;              // k-steps of q . k
  constexpr int KSV = kAttnBlock / F::KE;    // k-steps of p v
  constexpr int DTW = D / 64;
  constexpr int R = 16 * RT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lg = lane >> 4, lr = lane & 15;
  T* PB = reinterpret_cast<T*>(smem);                                  // [PARTS][R][VS]
  float* smax = reinterpret_cast<float*>(PB + F::PARTS * R * F::VS);   // [4][R]
  float* ssum = smax + 4 * R;                                          // [4][R]
  const int key0 = b * kAttnBlock;

  // s transposed for this wave's 16 keys: lane l holds keys 16 w + 4 (l / 16) + i
  // of query row 16 rt + l % 16
  float s[RT][4];
  {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      f4 acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = mma3<BF>(raw.k[ks], q[rt][ks], acc);
      const int pos = rq.L0 + min(16 * rt + lr, rq.W - 1);
#pragma unroll
      for (int i = 0; i < 4; ++i) s[rt][i] = key0 + 16 * wave + 4 * lg + i <= pos ? acc[i] * p.scale : -INFINITY;
    }
  }
  // block maximum per row: a lane's four keys, the four lanes of the row,
  // then the four waves in order
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float mx = fmaxf(fmaxf(fmaxf(s[rt][0], s[rt][1]), s[rt][2]), s[rt][3]);
    mx = swap_combine<false>(mx, FMax{});
    mx = swap_combine<true>(mx, FMax{});
    if (lg == 0) smax[wave * R + 16 * rt + lr] = mx;
  }
  __syncthreads();
  // p = exp(s - m_b) into LDS (row-major, (hi, lo)); its per-row sums
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = 16 * rt + lr;
    const float mb = fmaxf(fmaxf(fmaxf(smax[r], smax[R + r]), smax[2 * R + r]), smax[3 * R + r]);
    float pj[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pj[i] = mb == -INFINITY ? 0.0f : expf(s[rt][i] - mb);
    float sm = ((pj[0] + pj[1]) + pj[2]) + pj[3];
    sm = swap_combine<false>(sm, FAdd{});
    sm = swap_combine<true>(sm, FAdd{});
    if (lg == 0) ssum[wave * R + r] = sm;
    const int c = 16 * wave + 4 * lg;
    if constexpr (BF) {
      uint32_t hw[2], lw[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const uint16_t h0 = f2bf(pj[2 * t]), h1 = f2bf(pj[2 * t + 1]);
        hw[t] = h0 | ((uint32_t)h1 << 16);
        lw[t] = f2bf(pj[2 * t] - bf2f(h0)) | ((uint32_t)f2bf(pj[2 * t + 1] - bf2f(h1)) << 16);
      }
      *reinterpret_cast<uint2*>(PB + r * F::VS + c) = make_uint2(hw[0], hw[1]);
      *reinterpret_cast<uint2*>(PB + (R + r) * F::VS + c) = make_uint2(lw[0], lw[1]);
    } else {
      *reinterpret_cast<float4*>(PB + r * F::VS + c) = make_float4(pj[0], pj[1], pj[2], pj[3]);
    }
  }
  __syncthreads();   // ssum and P
  // the statistics of this lane's output rows 16 rt + 4 (l / 16) + i
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * rt + 4 * lg + i;
      out.m[rt][i] = fmaxf(fmaxf(fmaxf(smax[r], smax[R + r]), smax[2 * R + r]), smax[3 * R + r]);
      out.l[rt][i] = ((ssum[r] + ssum[R + r]) + ssum[2 * R + r]) + ssum[3 * R + r];
    }
  // acc_b = P V for this wave's dimension tiles
#pragma unroll
  for (int t = 0; t < DTW; ++t) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      f4 acc = f4{0.f, 0.f, 0.f, 0.f};
      const int r = 16 * rt + lr;
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) {
        const int c = F::KE * ks + F::PER * lg;
        Op2 a;
        a.h = *reinterpret_cast<const uint4*>(PB + r * F::VS + c);
        a.l = a.h;
        if constexpr (BF) a.l = *reinterpret_cast<const uint4*>(PB + (R + r) * F::VS + c);
        acc = mma3<BF>(a, raw.v[t][ks], acc);
      }
      out.acc[rt][t] = acc;
    }
  }
}

// Running attention state of this lane's rows (16 rt + 4 (lane / 16) + i)
// and dimensions (16 (w DTW + t) + lane % 16), in the layout of
// AttnBlockOut.
template <int RT, int DTW> struct AttnState {
  float M[RT][4], L[RT][4], A[RT][DTW][4];
};

// Merges a partial into the rows of st for which take(rt, i) holds;
// `first`: the partial starts those rows' state.
template <int RT, int DTW, class Take>
__device__ __forceinline__ void attn_state_merge(AttnState<RT, DTW>& st, const float (&m)[RT][4],
                                                 const float (&l)[RT][4], const float (&acc)[RT][DTW][4], bool first,
                                                 Take&& take) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (!take(rt, i)) continue;
      if (first) {
        st.M[rt][i] = m[rt][i];
        st.L[rt][i] = l[rt][i];
#pragma unroll
        for (int t = 0; t < DTW; ++t) st.A[rt][t][i] = acc[rt][t][i];
      } else {
        const MergeCoef k = attn_merge_coef(st.M[rt][i], st.L[rt][i], m[rt][i], l[rt][i]);
#pragma unroll
        for (int t = 0; t < DTW; ++t) st.A[rt][t][i] = attn_merge_acc(st.A[rt][t][i], acc[rt][t][i], k);
      }
    }
}

// Block b of span sp (first block b0) merged into st; rows before the
// block's first key are left as they are.  Synchronises the workgroup
// afterwards (the next block overwrites LDS).
template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_span_block(const AttnArgs& p, const ReqDesc& rq, int b, int b0,
                                                const Op2 (&q)[RT][D / AttnFmt<BF>::KE], const AttnRaw<BF, D>& raw,
                                                unsigned char* smem, AttnState<RT, D / 64>& st) {
  constexpr int DTW = D / 64;
  const int lane = threadIdx.x & 63;
  AttnBlockOut<BF, D, RT> o;
  attn_block<BF, D, RT>(p, rq, b, q, raw, smem, o);
  float acc[RT][DTW][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int t = 0; t < DTW; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[rt][t][i] = o.acc[rt][t][i];
  attn_state_merge<RT, DTW>(st, o.m, o.l, acc, b == b0, [&](int rt, int i) {
    return rq.L0 + min(16 * rt + 4 * (lane >> 4) + i, rq.W - 1) >= b * kAttnBlock;
  });
  __syncthreads();
}

// Blocks [b0, b1) of span sp = b0 / kAttnSpan.
__device__ __forceinline__ void attn_span_range(const ReqDesc& rq, int sp, int& b0, int& b1) {
  b0 = sp * kAttnSpan;
  b1 = min(b0 + kAttnSpan, (rq.L0 + rq.W - 1) / kAttnBlock + 1);
}

// Span `sp` of request rq for head h: its blocks merged in ascending order
// into st (a row's state starts at the span's first block).  The next
// block's keys and values are requested while the current one is computed.
template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_span(const AttnArgs& p, const ReqDesc& rq, int h, int sp,
                                          const Op2 (&q)[RT][D / AttnFmt<BF>::KE], unsigned char* smem,
                                          AttnState<RT, D / 64>& st) {
  int b0, b1;
  attn_span_range(rq, sp, b0, b1);
  // two buffers taken in turn: block b + 1 is requested before block b runs
  AttnRaw<BF, D> r0, r1;
  attn_fetch<BF, D>(p, rq, h, b0, r0);
  for (int b = b0; b < b1; b += 2) {
    if (b + 1 < b1) attn_fetch<BF, D>(p, rq, h, b + 1, r1);
    attn_span_block<BF, D, RT>(p, rq, b, b0, q, r0, smem, st);
    if (b + 1 >= b1) break;
    if (b + 2 < b1) attn_fetch<BF, D>(p, rq, h, b + 2, r0);
    attn_span_block<BF, D, RT>(p, rq, b + 1, b0, q, r1, smem, st);
  }
}

// Stores the span state of the rows of the request that reach span sp:
// pacc[sp][row][h][D] (A), pml[sp][row][h][2] (M, L), agent-scope stores.
template <int D, int RT>
__device__ __forceinline__ void attn_store_span(const AttnArgs& p, const ReqDesc& rq, int h, int sp,
                                                const AttnState<RT, D / 64>& st) {
  constexpr int DTW = D / 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * rt + 4 * (lane >> 4) + i;
      if (r < rq.W && rq.L0 + r >= sp * kAttnSpanKeys) {
        const size_t o = ((size_t)sp * p.part_rows + rq.row_start + r) * p.n_q + h;
#pragma unroll
        for (int t = 0; t < DTW; ++t)
          store_partial(p.pacc + o * D + 16 * (wave * DTW + t) + (lane & 15), st.A[rt][t][i]);
        if (wave == 0 && (lane & 15) < 2)
          store_partial(p.pml + o * 2 + (lane & 15), (lane & 15) ? st.L[rt][i] : st.M[rt][i]);
      }
    }
}

// Row r of request rq, head h: its span states (stored by attn_store_span,
// read with agent-scope loads) merged in ascending order, by one quarter
// wave (lane l % 16 holds dimensions [DQ (l % 16), DQ (l % 16) + DQ),
// DQ = D / 16); writes the attention output planes (OUT_COH: with
// agent-scope stores).
template <bool BF, int D, bool OUT_COH>
__device__ __forceinline__ void attn_merge_row(const AttnArgs& p, const ReqDesc& rq, int r, int h) {
  constexpr int DQ = D / 16;   // dimensions per lane
  constexpr int kB = 8;        // spans whose loads are in flight together
  static_assert(DQ % 4 == 0, "whole 16-byte reads per lane");
  const int ql = threadIdx.x & 15;
  const int row = rq.row_start + r;
  const int ns = (rq.L0 + r) / kAttnSpanKeys + 1;
  auto at = [&](int sp) { return ((size_t)sp * p.part_rows + row) * p.n_q + h; };
  const __amdgpu_buffer_rsrc_t racc = coherent_rsrc(p.pacc), rml = coherent_rsrc(p.pml);
  float M = 0.f, L = 0.f, A[DQ];
  for (int s0 = 0; s0 < ns; s0 += kB) {
    float ms[kB], ls[kB], as[kB][DQ];
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      const size_t o = at(min(s0 + u, ns - 1));   // past the last span: read it again, unused
      const float2 ml = ld_coherent2(rml, (uint32_t)(o * 2 * sizeof(float)));
      ms[u] = ml.x;
      ls[u] = ml.y;
#pragma unroll
      for (int t = 0; t < DQ; t += 4) {
        const float4 a = ld_coherent4(racc, (uint32_t)((o * D + DQ * ql + t) * sizeof(float)));
        as[u][t] = a.x;
        as[u][t + 1] = a.y;
        as[u][t + 2] = a.z;
        as[u][t + 3] = a.w;
      }
    }
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      if (s0 + u >= ns) break;
      if (s0 + u == 0) {
        M = ms[u];
        L = ls[u];
#pragma unroll
        for (int t = 0; t < DQ; ++t) A[t] = as[u][t];
      } else {
        const MergeCoef k = attn_merge_coef(M, L, ms[u], ls[u]);
#pragma unroll
        for (int t = 0; t < DQ; ++t) A[t] = attn_merge_acc(A[t], as[u][t], k);
      }
    }
  }
  float o[DQ];
#pragma unroll
  for (int t = 0; t < DQ; ++t) o[t] = A[t] / L;
  store_act_run<BF, OUT_COH, DQ>(p.out, p.out_plane, frag_index<BF>(row, h * D + DQ * ql, p.n_q * D), o);
}

}  // namespace as2d
