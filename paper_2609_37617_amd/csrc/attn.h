// Block-causal grouped-query attention of the verification step on matrix
// cores, shared by the per-operation kernels (kernels.hip) and the
// persistent step kernel (step.hip).
//
// Arithmetic of one row (position pos) and query head h, reading KV head
// g = floor(h n_kv / n_q).  Keys are taken in spans of kAttnSpanKeys = 128 at
// absolute positions, and a span in four chunks of kAttnChunk = 32 keys (one
// per wave); chunk c of span sp holds keys [128 sp + 32 c, 128 sp + 32 c + 32)
// up to pos:
//   s_j   = (q . k_j) * scale, a matrix-core product: for bf16 models q and
//           k are split into bf16 pairs (hi = bf16(x), lo = bf16(x - hi))
//           and s = q_hi k_hi + q_hi k_lo + q_lo k_hi over 32-wide k-steps;
//           float32 models use float32 products; scale = log2(e) / sqrt(d)
//           (rounded once to float32), so scores are in base-2 units;
//   m_c   = max_j s_j over the chunk;
//   p_j   = 2^(s_j - m_c), 0 for keys after pos (the hardware base-2
//           exponential, exp2 below: the same softmax as exp of the
//           natural-unit scores);
//   l_c   = sum_j p_j: a lane's keys of each 16-key tile in order, the two
//           tiles in order, then across lanes in a fixed butterfly;
//   acc_c = sum_j p_j v_j, a matrix-core product of the (hi, lo) splits of
//           p and v (p_hi v_hi + p_hi v_lo + p_lo v_hi) over the chunk.
// s is formed transposed (keys on the matrix-core rows), so each lane holds
// four consecutive keys of one query row per 16-key tile, and p stays in the
// registers that feed the p v product (bf16: the k-slice of lane group q is
// keys 4q .. 4q + 3 of the chunk's first tile and of its second tile, and v
// is read in that order).
// Merging a partial (m, l, acc) into a running state (M, L, A):
//   M' = max(M, m), a = exp2(M - M'), c = exp2(m - M'),
//   L = fma(L, a, l c), A = fma(A, a, acc c), M = M'.
// Two levels: the four chunks of a span are merged in ascending order,
// starting from the first; the spans' states are then merged in ascending
// order, starting from span 0.  The output is A / L.
//
// Every quantity of a row depends only on that row's query and the keys
// and values (matrix-core rows are independent), so a row gets the same
// bits whatever other rows share its tile and whoever merges its spans:
// the verification kernel (spans on different workgroups, span states
// through memory) or the prefill kernel (spans in a loop, in registers).
#pragma once
#include "tiles.h"

namespace as2d {

constexpr int kAttnChunk = kAttnSpanKeys / kWaves;   // keys of one wave's chunk of a span

// 2^x by the hardware instruction (0 for x = -inf).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

template <bool BF> struct AttnFmt {
  static constexpr int PER = BF ? 8 : 4;                  // elements per lane per k-step
  static constexpr int KE = 4 * PER;                      // k-step
  static constexpr int PARTS = BF ? 2 : 1;                // hi, lo planes
  static constexpr int KSV = kAttnChunk / KE;             // k-steps of p v over a chunk
};
static_assert(kAttnChunk == 32, "two 16-key tiles per chunk");

// Wave of a span group: four waves take a span's four chunks (a workgroup
// of eight waves runs two spans at once, one per group of four).
__device__ __forceinline__ int attn_wave() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & (kWaves - 1); }

// LDS of one span for RT row tiles: every wave's chunk sums acc_c
// [wave][rt][dimension tile][lane] (16 bytes per lane) and chunk statistics
// m_c, l_c [wave][16 RT] each.
template <bool BF, int D, int RT> __host__ __device__ constexpr int attn_span_lds_bytes() {
  return kWaves * RT * (D / 16) * 64 * 16 + 2 * kWaves * 16 * RT * 4;
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
  const MergeCoef k{exp2_hw(M - Mn), exp2_hw(m - Mn)};
  L = __builtin_fmaf(L, k.a, l * k.c);
  M = Mn;
  return k;
}
__device__ __forceinline__ float attn_merge_acc(float A, float acc, MergeCoef k) {
#pragma clang fp contract(off)
  return __builtin_fmaf(A, k.a, acc * k.c);
}

// The query rows of an attention block.  Block row rr (0 .. 16 RT) is the
// linear row u = u0 + rr of the query heads h0, h0 + 1, .. that share one KV
// head, u = (h - h0) W + i for request row i; rows past the n = heads x W of
// those heads repeat the last one (computed, never stored).  A block of one
// head: h0 = h, n = W, u0 = 0.  Each row's arithmetic is the same in any
// block.
struct AttnRows {
  int h0, W, n, u0;
  __device__ int lin(int rr) const { return min(u0 + rr, n - 1); }
  __device__ int head(int rr) const { return h0 + lin(rr) / W; }
  __device__ int row(int rr) const { return lin(rr) % W; }
  __device__ bool valid(int rr) const { return u0 + rr < n; }
};
__device__ __forceinline__ AttnRows attn_rows_of_head(int h, int W) { return AttnRows{h, W, W, 0}; }

// The operands of a block's queries: this lane's share of every k-step of
// row tiles rt < RT (block row 16 rt + lane % 16).
template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_load_q(const AttnArgs& p, const ReqDesc& rq, const AttnRows& rows,
                                            Op2 (&q)[RT][D / AttnFmt<BF>::KE]) {
  using F = AttnFmt<BF>;
  const int lane = threadIdx.x & 63;
  const int qcols = p.n_q * D;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int rr = 16 * rt + (lane & 15);
    const float4* base = reinterpret_cast<const float4*>(p.q + (size_t)(rq.row_start + rows.row(rr)) * qcols +
                                                         rows.head(rr) * D + F::PER * (lane >> 4));
#pragma unroll
    for (int ks = 0; ks < D / F::KE; ++ks) {
      float4 v[2];
      v[0] = ldg(base + F::KE / 4 * ks);
      if constexpr (BF) v[1] = ldg(base + F::KE / 4 * ks + 1);
      q[rt][ks] = split_op<BF>(v);
    }
  }
}

// One wave's chunk of keys and values as loaded from the cache (layout:
// AttnArgs), already the matrix-core operands.  k[kt]: the k-step slices of
// key 16 kt + l % 16 of the chunk (rows of the transposed product s).
// v[t][j]: dimension 16 t + l % 16 at the keys of k-step j of p v (bf16:
// keys 4 (l / 16) .. + 3 of both tiles; float32: keys 16 j + 4 (l / 16)
// .. + 3), in one 16-byte read per part (the V layout, AttnArgs).  Keys
// past the request's: K reads its last key (a branch-free load, never
// used); V is read as stored and its elements are set to zero where p v
// takes them (attn_v_operand: their p is 0, and 0 times a stale value must
// stay 0); a chunk that starts past the last key reads the last key's V
// block, all of it set to zero there.
template <bool BF, int D> struct AttnRaw {
  static constexpr int KS = D / AttnFmt<BF>::KE;   // k-steps of q . k
  static constexpr int DT = D / 16;                // dimension tiles
  static constexpr int KSV = AttnFmt<BF>::KSV;
  Op2 k[2][KS];
  Op2 v[DT][KSV];
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

// Wave w's chunk of span sp of KV head g.  Reads stay inside the slot's
// rows: K rows up to the last key, V blocks up to the last key's (the row
// stride is a multiple of 64, so a block ends inside the row).
// The keys (attn_fetch_k) and the values (attn_fetch_v) of the chunk.
template <bool BF, int D>
__device__ __forceinline__ void attn_fetch_k(const AttnArgs& p, const ReqDesc& rq, int g, int sp, AttnRaw<BF, D>& r) {
  using F = AttnFmt<BF>;
  using Raw = AttnRaw<BF, D>;
  using T = typename ET<BF>::T;
  const int wave = attn_wave(), lane = threadIdx.x & 63;
  const int lg = lane >> 4, lr = lane & 15;
  const int kc = sp * kAttnSpanKeys + kAttnChunk * wave;   // first key of the chunk
  const int last = rq.L0 + rq.W - 1;                       // last key of the request in this pass
  const size_t head = (size_t)rq.slot * p.slot_stride + (size_t)g * p.kv_cap * D;   // float32 units
  const T* kb = reinterpret_cast<const T*>(p.k_cache + head);
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const T* kr = kb + (size_t)min(kc + 16 * kt + lr, last) * F::PARTS * D + F::PER * lg;
#pragma unroll
    for (int ks = 0; ks < Raw::KS; ++ks) {
      r.k[kt][ks].h = ldg(reinterpret_cast<const uint4*>(kr + F::KE * ks));
      r.k[kt][ks].l = BF ? ldg(reinterpret_cast<const uint4*>(kr + D + F::KE * ks)) : r.k[kt][ks].h;
    }
  }
}
template <bool BF, int D>
__device__ __forceinline__ void attn_fetch_v(const AttnArgs& p, const ReqDesc& rq, int g, int sp, AttnRaw<BF, D>& r) {
  using F = AttnFmt<BF>;
  using Raw = AttnRaw<BF, D>;
  using T = typename ET<BF>::T;
  const int wave = attn_wave(), lane = threadIdx.x & 63;
  const int lg = lane >> 4, lr = lane & 15;
  const int kc = sp * kAttnSpanKeys + kAttnChunk * wave;   // first key of the chunk
  const int last = rq.L0 + rq.W - 1;                       // last key of the request in this pass
  const size_t head = (size_t)rq.slot * p.slot_stride + (size_t)g * p.kv_cap * D;   // float32 units
  const T* vb = reinterpret_cast<const T*>(p.v_cache + head);
  // the chunk's V block (v_elem): [parts][D][32]; a chunk past the last key
  // reads the last key's block instead (a branch-free load whose elements
  // attn_v_operand all sets to zero)
  const T* vc = vb + (size_t)(min(kc, last) >> 5) * F::PARTS * D * 32;
#pragma unroll
  for (int t = 0; t < Raw::DT; ++t) {
    const T* vr = vc + (16 * t + lr) * 32;
    if constexpr (BF) {
      // keys 4 lg .. 4 lg + 3 of the first tile, then of the second: columns
      // 8 lg .. 8 lg + 7 of the block (v_col)
      r.v[t][0] = Op2{ldg(reinterpret_cast<const uint4*>(vr + 8 * lg)),
                      ldg(reinterpret_cast<const uint4*>(vr + D * 32 + 8 * lg))};
    } else {
#pragma unroll
      for (int j = 0; j < Raw::KSV; ++j) {
        const uint4 o = ldg(reinterpret_cast<const uint4*>(vr + 16 * j + 4 * lg));
        r.v[t][j] = Op2{o, o};
      }
    }
  }
}
template <bool BF, int D>
__device__ __forceinline__ void attn_fetch(const AttnArgs& p, const ReqDesc& rq, int g, int sp, AttnRaw<BF, D>& r) {
  attn_fetch_k<BF, D>(p, rq, g, sp, r);
  attn_fetch_v<BF, D>(p, rq, g, sp, r);
}

// The V operand of dimension tile t and k-step j as p v takes it: elements
// of keys past the request's last key set to zero (a chunk past the last
// key holds the last key's block: all of it).  Done here rather than at the load, so that no wait
// for the data sits between the requests of the next chunk.
template <bool BF, int D>
__device__ __forceinline__ Op2 attn_v_operand(const AttnRaw<BF, D>& r, int t, int j, int kc, int last) {
  const int lg = (threadIdx.x & 63) >> 4;
  Op2 o = r.v[t][j];
  if (kc + kAttnChunk <= last + 1) return o;   // every key of the chunk is in the request
  if constexpr (BF) {
    const int n0 = min(max(last + 1 - (kc + 4 * lg), 0), 4);
    const int n1 = min(max(last + 1 - (kc + 16 + 4 * lg), 0), 4);
    const uint4 a = keep_first<true>(make_uint4(o.h.x, o.h.y, 0, 0), n0), b = keep_first<true>(make_uint4(o.h.z, o.h.w, 0, 0), n1);
    const uint4 c = keep_first<true>(make_uint4(o.l.x, o.l.y, 0, 0), n0), d = keep_first<true>(make_uint4(o.l.z, o.l.w, 0, 0), n1);
    o.h = make_uint4(a.x, a.y, b.x, b.y);
    o.l = make_uint4(c.x, c.y, d.x, d.y);
  } else {
    o.h = keep_first<false>(o.h, min(max(last + 1 - (kc + 16 * j + 4 * lg), 0), 4));
    o.l = o.h;
  }
  return o;
}

// Running attention state of this lane's rows (16 rt + 4 (lane / 16) + i)
// and dimensions (16 (w DTW + t) + lane % 16).
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

// The state of span sp for the block rows of row tiles rt < RT (queries q;
// this wave's chunk of keys and values in raw), in the layout of AttnState:
// for lane l and i < 4, block row 16 rt + 4 (l / 16) + i, dimensions
// 16 (w DTW + t) + l % 16.  Rows whose position is before the span's first
// key get no meaningful state (they are never stored or merged).  Four waves
// (a span group, attn_wave);
// smem: attn_span_lds_bytes<BF, D, RT>(), not in use on entry (the caller
// synchronises the workgroup before it is written again).  Two steps:
// attn_span_chunks (each wave's chunk sums into the LDS; q and raw are not
// needed after it) and attn_merge_chunks.
struct NoOp {
  __device__ void operator()() const {}
};
template <bool BF, int D, int RT, class PreV = NoOp>
__device__ __forceinline__ void attn_span_chunks(const AttnArgs& p, const ReqDesc& rq, const AttnRows& rows, int sp,
                                                 const Op2 (&q)[RT][D / AttnFmt<BF>::KE], const AttnRaw<BF, D>& raw,
                                                 unsigned char* smem, PreV pre_v = PreV{}) {
#pragma clang fp contract(off)
  using Raw = AttnRaw<BF, D>;
  constexpr int KS = Raw::KS, DT = Raw::DT, DTW = D / 64, R = 16 * RT;
  const int wave = attn_wave(), lane = threadIdx.x & 63;
  const int lg = lane >> 4, lr = lane & 15;
  const int kc = sp * kAttnSpanKeys + kAttnChunk * wave;
  const int last = rq.L0 + rq.W - 1;   // last key of the request in this pass
  // every key of the chunk is in the request (wave-uniform): p v takes the
  // values as loaded, without the masking path's copies
  const bool whole = kc + kAttnChunk <= last + 1;
  f4* SA = reinterpret_cast<f4*>(smem);                                 // [wave][rt][t][lane]
  float* SM = reinterpret_cast<float*>(SA + kWaves * RT * DT * 64);   // [wave][R]
  float* SL = SM + kWaves * R;                                          // [wave][R]

  // s of every row tile first, so that the keys are free before p v
  float s[RT][2][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    // s transposed: lane l holds keys kc + 16 kt + 4 (l / 16) + i of block row 16 rt + l % 16
    const int pos = rq.L0 + rows.row(16 * rt + lr);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      f4 acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = mma3<BF>(raw.k[kt][ks], q[rt][ks], acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) s[rt][kt][i] = kc + 16 * kt + 4 * lg + i <= pos ? acc[i] * p.scale : -INFINITY;
    }
  }
  pre_v();   // a caller that fetches the values only now (the keys' registers are free)
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float mx = s[rt][0][0];
#pragma unroll
    for (int e = 1; e < 8; ++e) mx = fmaxf(mx, s[rt][e >> 2][e & 3]);
    mx = swap_combine<false>(mx, FMax{});
    mx = swap_combine<true>(mx, FMax{});
    float pj[2][4];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) pj[kt][i] = mx == -INFINITY ? 0.0f : exp2_hw(s[rt][kt][i] - mx);
    float sm = (((pj[0][0] + pj[0][1]) + pj[0][2]) + pj[0][3]) + (((pj[1][0] + pj[1][1]) + pj[1][2]) + pj[1][3]);
    sm = swap_combine<false>(sm, FAdd{});
    sm = swap_combine<true>(sm, FAdd{});
    if (lg == 0) {
      SM[wave * R + 16 * rt + lr] = mx;
      SL[wave * R + 16 * rt + lr] = sm;
    }
    // acc_c = p v for every dimension tile, p straight from registers
    f4* sa = SA + (size_t)(wave * RT + rt) * DT * 64 + lane;
    if constexpr (BF) {
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {   // elements 2 w, 2 w + 1: tile w / 2, keys 2 (w % 2), 2 (w % 2) + 1
        const float v0 = pj[w >> 1][2 * (w & 1)], v1 = pj[w >> 1][2 * (w & 1) + 1];
        const uint16_t h0 = f2bf(v0), h1 = f2bf(v1);
        hw[w] = h0 | ((uint32_t)h1 << 16);
        lw[w] = f2bf(v0 - bf2f(h0)) | ((uint32_t)f2bf(v1 - bf2f(h1)) << 16);
      }
      const Op2 a{make_uint4(hw[0], hw[1], hw[2], hw[3]), make_uint4(lw[0], lw[1], lw[2], lw[3])};
      if (whole) {
#pragma unroll
        for (int t = 0; t < DT; ++t) sa[t * 64] = mma3<BF>(a, raw.v[t][0], f4{0.f, 0.f, 0.f, 0.f});
      } else {
#pragma unroll
        for (int t = 0; t < DT; ++t) sa[t * 64] = mma3<BF>(a, attn_v_operand<BF, D>(raw, t, 0, kc, last), f4{0.f, 0.f, 0.f, 0.f});
      }
    } else {
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        f4 acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const uint4 a = make_uint4(__float_as_uint(pj[kt][0]), __float_as_uint(pj[kt][1]), __float_as_uint(pj[kt][2]),
                                     __float_as_uint(pj[kt][3]));
          acc = mma_step<false>(a, whole ? raw.v[t][kt].h : attn_v_operand<BF, D>(raw, t, kt, kc, last).h, acc);
        }
        sa[t * 64] = acc;
      }
    }
  }
}

template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_merge_chunks(unsigned char* smem, AttnState<RT, D / 64>& st) {
#pragma clang fp contract(off)
  constexpr int DT = D / 16, DTW = D / 64, R = 16 * RT;
  const int wave = attn_wave(), lane = threadIdx.x & 63, lg = lane >> 4;
  const f4* SA = reinterpret_cast<const f4*>(smem);                          // [wave][rt][t][lane]
  const float* SM = reinterpret_cast<const float*>(SA + kWaves * RT * DT * 64);   // [wave][R]
  const float* SL = SM + kWaves * R;                                              // [wave][R]
  lds_sync();   // LDS only: global loads in flight (the next span's) stay in flight
  // the four chunks merged in order, for this wave's dimension tiles
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    MergeCoef k[kWaves - 1][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * rt + 4 * lg + i;
      float M = SM[r], L = SL[r];
#pragma unroll
      for (int c = 1; c < kWaves; ++c) k[c - 1][i] = attn_merge_coef(M, L, SM[c * R + r], SL[c * R + r]);
      st.M[rt][i] = M;
      st.L[rt][i] = L;
    }
#pragma unroll
    for (int tw = 0; tw < DTW; ++tw) {
      const int t = wave * DTW + tw;
      f4 A = SA[(size_t)(0 * RT + rt) * DT * 64 + t * 64 + lane];
#pragma unroll
      for (int c = 1; c < kWaves; ++c) {
        const f4 a = SA[(size_t)(c * RT + rt) * DT * 64 + t * 64 + lane];
#pragma unroll
        for (int i = 0; i < 4; ++i) A[i] = attn_merge_acc(A[i], a[i], k[c - 1][i]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) st.A[rt][tw][i] = A[i];
    }
  }
}

template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_span_state(const AttnArgs& p, const ReqDesc& rq, const AttnRows& rows, int sp,
                                                const Op2 (&q)[RT][D / AttnFmt<BF>::KE], const AttnRaw<BF, D>& raw,
                                                unsigned char* smem, AttnState<RT, D / 64>& st) {
  attn_span_chunks<BF, D, RT>(p, rq, rows, sp, q, raw, smem);
  attn_merge_chunks<BF, D, RT>(smem, st);
}

// KV head of the query heads of a block.
__device__ __forceinline__ int attn_kv_head(const AttnArgs& p, const AttnRows& rows) { return rows.h0 * p.n_kv / p.n_q; }

// Span sp of request rq for a block's rows: fetch, then attn_span_state.
template <bool BF, int D, int RT>
__device__ __forceinline__ void attn_span(const AttnArgs& p, const ReqDesc& rq, const AttnRows& rows, int sp,
                                          const Op2 (&q)[RT][D / AttnFmt<BF>::KE], unsigned char* smem,
                                          AttnState<RT, D / 64>& st) {
  AttnRaw<BF, D> raw;
  attn_fetch<BF, D>(p, rq, attn_kv_head(p, rows), sp, raw);
  attn_span_state<BF, D, RT>(p, rq, rows, sp, q, raw, smem, st);
}

// Stores the span state of the block's rows that reach span sp:
// pacc[row][h][sp][D] (A), pml[row][h][sp][2] (M, L), agent-scope stores.
template <int D, int RT>
__device__ __forceinline__ void attn_store_span(const AttnArgs& p, const ReqDesc& rq, const AttnRows& rows, int sp,
                                                const AttnState<RT, D / 64>& st) {
  constexpr int DTW = D / 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = 16 * rt + 4 * (lane >> 4) + i;
      const int r = rows.row(rr);
      if (rows.valid(rr) && rq.L0 + r >= sp * kAttnSpanKeys) {
        const size_t o = ((size_t)(rq.row_start + r) * p.n_q + rows.head(rr)) * p.part_spans + sp;
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
  auto at = [&](int sp) { return ((size_t)row * p.n_q + h) * p.part_spans + sp; };
  const __amdgpu_buffer_rsrc_t racc = coherent_rsrc(p.pacc), rml = coherent_rsrc(p.pml);
  float M = 0.f, L = 0.f, A[DQ];
  // batches of kB spans; the next batch is requested before the current one
  // is merged (past the last span: the last one again, unused)
  struct Batch {
    float m[kB], l[kB], a[kB][DQ];
  };
  auto load = [&](int s0, Batch& b) {
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      const size_t o = at(min(s0 + u, ns - 1));
      const float2 ml = ld_coherent2(rml, (uint32_t)(o * 2 * sizeof(float)));
      b.m[u] = ml.x;
      b.l[u] = ml.y;
#pragma unroll
      for (int t = 0; t < DQ; t += 4) {
        const float4 a = ld_coherent4(racc, (uint32_t)((o * D + DQ * ql + t) * sizeof(float)));
        b.a[u][t] = a.x;
        b.a[u][t + 1] = a.y;
        b.a[u][t + 2] = a.z;
        b.a[u][t + 3] = a.w;
      }
    }
  };
  auto merge = [&](int s0, const Batch& b) {
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      if (s0 + u >= ns) break;
      if (s0 + u == 0) {
        M = b.m[u];
        L = b.l[u];
#pragma unroll
        for (int t = 0; t < DQ; ++t) A[t] = b.a[u][t];
      } else {
        const MergeCoef k = attn_merge_coef(M, L, b.m[u], b.l[u]);
#pragma unroll
        for (int t = 0; t < DQ; ++t) A[t] = attn_merge_acc(A[t], b.a[u][t], k);
      }
    }
  };
  Batch b0, b1;
  load(0, b0);
  for (int s0 = 0; s0 < ns; s0 += 2 * kB) {
    if (s0 + kB < ns) load(s0 + kB, b1);
    merge(s0, b0);
    if (s0 + kB >= ns) break;
    if (s0 + 2 * kB < ns) load(s0 + 2 * kB, b0);
    merge(s0 + kB, b1);
  }
  float o[DQ];
#pragma unroll
  for (int t = 0; t < DQ; ++t) o[t] = A[t] / L;
  store_act_run<BF, OUT_COH, DQ>(p.out, p.out_plane, frag_index<BF>(row, h * D + DQ * ql, p.n_q * D), o);
}

// Row i of request rq, head h, by one wave: the same fold as attn_merge_row
// (span states in ascending order from span 0), with lane l holding
// dimensions [DL l, DL l + DL), DL = D / 64.  The states come in batches of
// kB spans, the next batch requested before the current one is folded; the
// fold's coefficients of a batch are computed one span per lane: the
// running maximum before span s is the maximum of m over spans 0 .. s - 1,
// which a prefix scan gives exactly (fmax rounds nothing).  The states were
// stored by an earlier kernel; the output planes are read by a later one.
template <bool BF, int D>
__device__ __forceinline__ void attn_merge_wave(const AttnArgs& p, const ReqDesc& rq, int i, int h) {
#pragma clang fp contract(off)
  constexpr int DL = D / 64;   // dimensions per lane
  constexpr int kB = 16;       // spans per batch
  static_assert(DL == 1 || DL == 2, "64 or 128 dimensions");
  const int lane = threadIdx.x & 63, bl = lane & (kB - 1);
  const int row = rq.row_start + i;
  const int ns = (rq.L0 + i) / kAttnSpanKeys + 1;
  auto at = [&](int sp) { return ((size_t)row * p.n_q + h) * p.part_spans + sp; };
  struct Batch {
    float m, l, a[kB][DL];
  };
  // past the last span: the last one again, unused
  auto load = [&](int s0, Batch& b) {
    const float2 ml = ldg(reinterpret_cast<const float2*>(p.pml + at(min(s0 + bl, ns - 1)) * 2));
    b.m = ml.x;
    b.l = ml.y;
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      const float* src = p.pacc + at(min(s0 + u, ns - 1)) * D + DL * lane;
      if constexpr (DL == 2) {
        const float2 v = ldg(reinterpret_cast<const float2*>(src));
        b.a[u][0] = v.x;
        b.a[u][1] = v.y;
      } else {
        b.a[u][0] = ldg(src);
      }
    }
  };
  float M = -INFINITY, L = 0.f, A[DL];
  auto merge = [&](int s0, const Batch& b) {
    // lane u: the running maximum after span s0 + u (mx) and before it (mb)
    float mx = s0 + bl < ns ? b.m : -INFINITY;
#pragma unroll
    for (int d = 1; d < kB; d <<= 1) {
      const float o = __shfl_up(mx, d, kB);
      if (bl >= d) mx = fmaxf(mx, o);
    }
    mx = fmaxf(M, mx);
    float mb = __shfl_up(mx, 1, kB);
    if (bl == 0) mb = M;
    const float ca = exp2_hw(mb - mx), cc = exp2_hw(b.m - mx);
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      if (s0 + u < ns) {
        const float lu = lane_value(b.l, u);
        if (s0 + u == 0) {
          L = lu;
#pragma unroll
          for (int t = 0; t < DL; ++t) A[t] = b.a[u][t];
        } else {
          const float ka = lane_value(ca, u), kc = lane_value(cc, u);
          L = __builtin_fmaf(L, ka, lu * kc);
#pragma unroll
          for (int t = 0; t < DL; ++t) A[t] = __builtin_fmaf(A[t], ka, b.a[u][t] * kc);
        }
      }
    }
    M = lane_value(mx, min(ns - s0, kB) - 1);
  };
  Batch b0, b1;
  load(0, b0);
  for (int s0 = 0; s0 < ns; s0 += 2 * kB) {
    if (s0 + kB < ns) load(s0 + kB, b1);
    merge(s0, b0);
    if (s0 + kB >= ns) break;
    if (s0 + 2 * kB < ns) load(s0 + 2 * kB, b0);
    merge(s0 + kB, b1);
  }
  float o[DL];
#pragma unroll
  for (int t = 0; t < DL; ++t) o[t] = A[t] / L;
  const size_t e = frag_index<BF>(row, h * D + DL * lane, p.n_q * D);
  if constexpr (DL == 2) store_act_run<BF, false, 2>(p.out, p.out_plane, e, o);
  else store_act<BF, false>(p.out, p.out_plane, e, o[0]);
}

}  // namespace as2d
