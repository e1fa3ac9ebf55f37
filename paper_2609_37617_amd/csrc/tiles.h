// Tile-level device functions of the verification step, shared by the
// per-operation kernels (kernels.hip) and the persistent step kernel
// (step.hip), so both compute every row bit for bit alike.
//
// COH (template flag): true when the outputs are read by other workgroups
// of the same kernel (persistent step kernel), see st<COH> in common.h.
#pragma once
#include "common.h"

namespace as2d {

// ---------------------------------------------------------------------------
// Embedding gather of row m: residual x (float32) from a token embedding or
// an audio staging row, the planes of x * g for the first RMSNorm (gain g),
// and the row's sum-of-squares partials per 32-column pair.  256 threads;
// srow: LDS scratch of H floats.

template <bool BF, bool COH>
__device__ __forceinline__ void embed_row(const RowDesc* __restrict__ rows, int m, const typename ET<BF>::T* __restrict__ embed,
                          const typename ET<BF>::T* __restrict__ audio, int H, const float* __restrict__ gain,
                          float* __restrict__ x, float* __restrict__ sumsq, void* __restrict__ xg,
                          long long xg_plane, float* srow) {
  using T = typename ET<BF>::T;
  constexpr int kPer = 8, kPasses = 4;   // H <= 256 * 8 * 4
  const RowDesc rd = load_invariant(rows + m);
  const T* src = rd.token >= 0 ? embed + (size_t)rd.token * H : audio + (size_t)rd.src * H;
  float v[kPasses][kPer];
#pragma unroll
  for (int ps = 0; ps < kPasses; ++ps) {
    const int c0 = (ps * 256 + threadIdx.x) * kPer;
    if (c0 < H) {
      if constexpr (BF) {
        const uint4 u = *reinterpret_cast<const uint4*>(src + c0);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[ps][2 * t] = bf2f(w[t] & 0xffffu);
          v[ps][2 * t + 1] = bf2f(w[t] >> 16);
        }
      } else {
        const float4 a = *reinterpret_cast<const float4*>(src + c0);
        const float4 b = *reinterpret_cast<const float4*>(src + c0 + 4);
        v[ps][0] = a.x; v[ps][1] = a.y; v[ps][2] = a.z; v[ps][3] = a.w;
        v[ps][4] = b.x; v[ps][5] = b.y; v[ps][6] = b.z; v[ps][7] = b.w;
      }
    }
  }
#pragma unroll
  for (int ps = 0; ps < kPasses; ++ps) {
    const int c0 = (ps * 256 + threadIdx.x) * kPer;
    if (c0 < H) {
#pragma unroll
      for (int t = 0; t < kPer; ++t) {
        st<COH>(x + (size_t)m * H + c0 + t, v[ps][t]);
        store_act<BF, COH>(xg, xg_plane, frag_index<BF>(m, c0 + t, H), v[ps][t] * gain[c0 + t]);
        srow[c0 + t] = v[ps][t];
      }
    }
  }
  lds_sync();
  // one pair per half-wave
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n_pairs = H / kPairCols;
  for (int u0 = wave * 2; u0 < n_pairs; u0 += 8) {
    const int g = u0 + (lane >> 5);
    const float e = g < n_pairs ? srow[g * kPairCols + (lane & 31)] : 0.0f;
    const float s = half_sum(e * e);
    if ((lane & 31) == 0 && g < n_pairs) st<COH>(sumsq + (size_t)m * n_pairs + g, s);
  }
}

// ---------------------------------------------------------------------------
// Fused GEMM epilogues over rows [r0, r1) of `np` consecutive tile pairs
// starting at pair `pair0`; F holds their finished values (float32, row
// stride fs, pair pp at columns [32 pp, 32 pp + 32)).  NTH threads.  Every
// per-pair sum runs on one half-wave in a fixed pattern, and the per-pair
// arg-max is exact, so a row's results do not depend on how many pairs or
// rows the call covers.

template <bool BF, int EPI, bool COH, int NTH = 256>
__device__ __forceinline__ void epilogue_rows(const GemmArgs& p, float* F, int fs, int pair0, int np, int r0, int r1) {
  constexpr int kUnits = NTH / 32;              // (row, pair) units per pass: one per half-wave
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int N = p.N, C = np * kPairCols;
  const int n0 = pair0 * kPairCols;
  const int units = (r1 - r0) * np;           // (row, pair) units of the reductions
  if constexpr (EPI == EPI_RESID || EPI == EPI_DOWN) {
    // x_out = x + Y; planes of x_out * g for the next RMSNorm; sum of squares
    for (int idx = tid; idx < (r1 - r0) * C; idx += NTH) {
      const int m = r0 + idx / C, c = idx % C;
      const int n = n0 + c;
      const size_t o = (size_t)m * N + n;
      const float v = ldg(p.x + o) + F[(m - r0) * fs + c];
      st<COH>(p.x_out + o, v);
      store_act<BF, COH>(p.out, p.out_plane, frag_index<BF>(m, n, N), v * ldg(p.gain_next + n));
      F[(m - r0) * fs + c] = v;
    }
    lds_sync();
    for (int u0 = wave * 2; u0 < units; u0 += kUnits) {
      const int u = u0 + (lane >> 5);
      const bool ok = u < units;
      const int m = ok ? r0 + u / np : r0, pp = u % np;
      const float e = ok ? F[(m - r0) * fs + pp * kPairCols + (lane & 31)] : 0.0f;
      const float s = half_sum(e * e);
      if ((lane & 31) == 0 && ok) st<COH>(p.sumsq_out + (size_t)m * (N / kPairCols) + pair0 + pp, s);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // pair g: gate columns 16 g .. 16 g + 15 (tile 0), the same up columns (tile 1)
    const int F2 = N / 2;
    for (int idx = tid; idx < (r1 - r0) * np * 16; idx += NTH) {
      const int m = r0 + idx / (np * 16), r = idx % (np * 16);
      const int pp = r >> 4, c = r & 15;
      const float g = F[(m - r0) * fs + pp * kPairCols + c], u = F[(m - r0) * fs + pp * kPairCols + 16 + c];
      store_act<BF, COH>(p.out, p.out_plane, frag_index<BF>(m, (pair0 + pp) * 16 + c, F2),
                         g / (1.0f + expf(-g)) * u);
    }
  } else if constexpr (EPI == EPI_QKV) {
    // PACK_ROPE_PAIRS: pair q of a head holds dims 16 q + c (tile 0) and
    // d/2 + 16 q + c (tile 1), the two halves RoPE rotates together
    const int d = p.head_dim, half = d >> 1, ppd = d / kPairCols;
    for (int idx = tid; idx < (r1 - r0) * C; idx += NTH) {
      const int m = r0 + idx / C, c = idx % C;
      const int pair = pair0 + c / kPairCols, j = (c >> 4) & 1, cc = c & 15;
      const int head = pair / ppd, q = pair % ppd;
      const int i = 16 * q + cc;                 // rotation index
      const int dd = j * half + i;               // dimension within the head
      const int n = head * d + dd;               // original output column
      const RowDesc rd = load_invariant(p.rows + m);
      const float* Fr = F + (m - r0) * fs;
      float v = Fr[c] + (p.bias ? ldg(p.bias + n) : 0.0f);
      if (head < p.n_q + p.n_kv) {
        const int pn = j ? n - half : n + half;
        const float partner = Fr[c ^ 16] + (p.bias ? ldg(p.bias + pn) : 0.0f);
        const float cs = ldg(p.rope_cs + ((size_t)rd.pos * half + i) * 2);
        const float sn = ldg(p.rope_cs + ((size_t)rd.pos * half + i) * 2 + 1);
        v = j == 0 ? v * cs - partner * sn : v * cs + partner * sn;
        if (head < p.n_q) {
          st<COH>(p.q_out + (size_t)m * p.n_q * d + n, v);
        } else {
          // K: [pos][(hi, lo)][d] (bf16) or [pos][d] (float32), see AttnArgs
          const int kvh = head - p.n_q;
          float* kb = p.k_cache + (size_t)rd.slot * p.slot_stride + (size_t)kvh * p.kv_cap * d;
          if constexpr (BF) {
            uint16_t* k16 = reinterpret_cast<uint16_t*>(kb) + (size_t)rd.pos * 2 * d + dd;
            const uint16_t hi = f2bf(v);
            st<COH>(k16, hi);
            st<COH>(k16 + d, f2bf(v - bf2f(hi)));
          } else {
            st<COH>(kb + (size_t)rd.pos * d + dd, v);
          }
        }
      } else {
        // V: blocks of 32 positions (v_elem, see AttnArgs)
        const int kvh = head - p.n_q - p.n_kv;
        float* vb = p.v_cache + (size_t)rd.slot * p.slot_stride + (size_t)kvh * p.kv_cap * d;
        if constexpr (BF) {
          uint16_t* v16 = reinterpret_cast<uint16_t*>(vb);
          const uint16_t hi = f2bf(v);
          st<COH>(v16 + v_elem(rd.pos, 0, dd, d, true), hi);
          st<COH>(v16 + v_elem(rd.pos, 1, dd, d, true), f2bf(v - bf2f(hi)));
        } else {
          st<COH>(vb + v_elem(rd.pos, 0, dd, d, false), v);
        }
      }
    }
  } else {  // EPI_ARGMAX (identity column order: column = token id)
    // one (row, pair) per thread: the largest value, the lowest column
    // among equal values and the second-largest value (equal to the
    // largest when two columns tie); exact, so the order of the scan is
    // immaterial.  A non-finite value makes the pair's partial NaN.
    for (int u = tid; u < units; u += NTH) {
      const int m = r0 + u / np, pp = u % np;
      const int n0p = (pair0 + pp) * kPairCols;
      const float* Fr = F + (m - r0) * fs + pp * kPairCols;
      float best = Fr[0], second = -INFINITY;
      int bi = n0p;
      bool bad = !isfinite(best);
      if (p.logits) p.logits[(size_t)m * N + n0p] = best;   // read by the host only
      for (int c = 1; c < kPairCols; ++c) {
        const float v = Fr[c];
        if (p.logits) p.logits[(size_t)m * N + n0p + c] = v;
        bad |= !isfinite(v);
        if (v > best) {
          second = best;
          best = v;
          bi = n0p + c;
        } else {
          second = fmaxf(second, v);
        }
      }
      const size_t o = (size_t)m * (N / kPairCols) + pair0 + pp;
      st<COH>(p.amax_val + o, bad ? __builtin_nanf("") : best);
      st<COH>(p.amax_val2 + o, second);
      st<COH>(p.amax_idx + o, bi);
    }
  }
}

// ---------------------------------------------------------------------------
// Split-K fixup, shared by both GEMM paths: the workgroup that finishes
// tile `tile` last sums, for each of its output elements (rows < M, columns
// [n0, n0 + C)), the KS split partials in split order, scales row m by
// s_scale[m] (A_NORM) and writes the result to F (row stride fs, rows from
// r0).  Loads are issued in batches across elements and splits.

template <int AM, int NTH = 256>
__device__ __forceinline__ void fixup_rows(const GemmArgs& p, int M, int n0, int C, int r0, int r1, const float* s_scale,
                           float* F, int fs) {
  constexpr int kEl = 2;   // elements per thread per batch (kEl x kMaxSplits loads in flight)
  const int E = (r1 - r0) * C;
  for (int e0 = threadIdx.x; e0 < E; e0 += NTH * kEl) {
    float v[kEl][kMaxSplits];
#pragma unroll
    for (int t = 0; t < kEl; ++t) {
      const int e = e0 + t * NTH;
      const int m = r0 + e / C, c = e % C;
#pragma unroll
      for (int sp = 0; sp < kMaxSplits; ++sp)
        if (e < E && sp < p.KS) v[t][sp] = load_partial(&p.part[((size_t)sp * M + m) * p.N + n0 + c]);
    }
#pragma unroll
    for (int t = 0; t < kEl; ++t) {
      const int e = e0 + t * NTH;
      if (e < E) {
        const int m = r0 + e / C, c = e % C;
        float sum = v[t][0];
#pragma unroll
        for (int sp = 1; sp < kMaxSplits; ++sp)
          if (sp < p.KS) sum += v[t][sp];
        F[(m - r0) * fs + c] = AM == A_NORM ? sum * s_scale[m] : sum;
      }
    }
  }
}

// Slice q of ns of the k-range [kt0, kt0 + n): [kt0 + q n / ns, kt0 + (q + 1) n / ns).
__device__ __forceinline__ int slice_start(int kt0, int n, int q, int ns) { return kt0 + (q * n) / ns; }

// Publishes a workgroup's split partials for (rows < M, columns [n0, n0 + C))
// given by `val(m, c)` and returns true in the workgroup that arrives last
// at counter `cnt` (it then resets the counter for the next launch).
template <int NTH = 256, class Val>
__device__ __forceinline__ bool publish_split(const GemmArgs& p, int M, int split, int n0, int C, int* cnt, int* s_flag, Val&& val) {
  for (int e = threadIdx.x; e < M * C; e += NTH) {
    const int m = e / C, c = e % C;
    store_partial(&p.part[((size_t)split * M + m) * p.N + n0 + c], val(m, c));
  }
  wait_vmem();
  __syncthreads();  // every wave's partial stores are performed
  if (threadIdx.x == 0) *s_flag = counter_add(cnt, 1) == p.KS - 1;
  __syncthreads();
  if (!*s_flag) return false;
  if (threadIdx.x == 0) st<true>(cnt, 0);  // ready for the next launch
  return true;
}

// Row scales 1 / sqrt(mean(x^2) + eps) of an A_NORM GEMM for rows [0, M)
// into s_scale, from the rows' per-pair sum-of-squares partials (at most
// 256 pairs: hidden <= 8192).  Each row is summed in a fixed pattern (lane
// l: partials l, l + 64, ...; then a butterfly), so its value depends on
// the row alone; wave w of NW takes rows w, w + NW, ..., eight rows per
// batch with all their loads in flight together.
template <int AM, int NW = kWaves>
__device__ __forceinline__ void row_scales(const GemmArgs& p, int M, float* s_scale) {
  if constexpr (AM == A_NORM) {
    constexpr int kR = 8, kT = 4;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int np = p.n_norm_pairs;
    for (int m0 = wave; m0 < M; m0 += NW * kR) {
      float s[kR];
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const int m = m0 + NW * r;
        s[r] = 0.0f;
#pragma unroll
        for (int t = 0; t < kT; ++t)
          if (m < M && lane + 64 * t < np) s[r] += p.sumsq[(size_t)m * np + lane + 64 * t];
      }
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const int m = m0 + NW * r;
        const float tot = wave_sum(s[r]);
        if (lane == 0 && m < M) s_scale[m] = 1.0f / sqrtf(tot / (float)p.K + p.eps);
      }
    }
  }
}

// row_scales in two steps for the direct paths, with the same sums (the
// same bits): row_scale_loads reads the sum-of-squares partials of this
// wave's rows m = wave + NW r (r < RPW) with no branch around the loads
// and forms each lane's partial sum; it is called right after the first
// weight loads, so its wait is one the stream needs anyway.
// row_scale_finish adds the lanes (same butterfly) for the rows < M and
// writes s_scale; it runs after the stream.
template <int AM, int RPW, int NW = kWaves>
__device__ __forceinline__ void row_scale_loads(const GemmArgs& p, int M, float (&s)[RPW]) {
  if constexpr (AM == A_NORM) {
    constexpr int kT = 4;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int np = p.n_norm_pairs;
    float v[RPW][kT];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int m = wave + NW * r, mm = m < M ? m : 0;
#pragma unroll
      for (int t = 0; t < kT; ++t) {
        const int i = lane + 64 * t;
        v[r][t] = ldg(p.sumsq + (size_t)mm * np + (i < np ? i : 0));
      }
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      s[r] = 0.0f;
#pragma unroll
      for (int t = 0; t < kT; ++t)
        if (wave + NW * r < M && lane + 64 * t < np) s[r] += v[r][t];
    }
  }
}
template <int AM, int RPW, int NW = kWaves>
__device__ __forceinline__ void row_scale_finish(const GemmArgs& p, int M, const float (&s)[RPW], float* s_scale) {
  if constexpr (AM == A_NORM) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int m = wave + NW * r;
      if (m < M) {
        const float tot = wave_sum(s[r]);
        if (lane == 0) s_scale[m] = 1.0f / sqrtf(tot / (float)p.K + p.eps);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// GEMM tiles.  Every output element is summed in one order whatever the
// path, the tile shape or the number of rows: k-split s of the plan
// (splits in order), in ns slices (slice_start, in order; ns from the
// plan), each slice accumulated over its k-steps in order by MFMA from
// zero; then (((q0 + q1) + q2) + ...) over the slices of a split and the
// splits added in order.  A row's result therefore depends on the matrix
// shape alone, never on the rows that share the pass or the kernel that
// computes it.
//
// Direct path (up to kDirectMT row tiles): a workgroup of NW waves owns NP
// tile pairs (32 NP columns) of one split; wave w streams the ns / NW
// consecutive slices [w ns / NW, (w + 1) ns / NW) of the split for all NP
// pairs as one contiguous run of k-steps, with the activation fragments
// (one per k-step, shared by the NP pairs) loaded straight from the planes;
// each slice's sums go to LDS and the slices meet there.  `wait()` is
// called after the first weight loads are issued and before any activation
// is read (the persistent kernel waits there for the producer of A).
// Returns true when this workgroup finished its pairs (ran their
// epilogue).
//   smem: dynamic LDS of gemm_direct_lds_bytes<MT, NP>(ns); s_scale:
//   kMaxRows floats; s_flag: one int.

template <int MT, int NP> __host__ __device__ constexpr int gemm_direct_lds_bytes(int ns) {
  return (ns * MT * NP * 512 + 16 * MT * (NP * kPairCols + 1)) * 4;
}
// k-steps in flight per wave.  Shallow: as many as about 96 registers hold
// (several workgroups per compute unit).  Deep: about 200 registers (one
// workgroup per compute unit); the last round of a wave re-reads its last
// k-step P times, so depth only pays on long runs of k-steps.
template <int MT, int NP, bool DEEP> __host__ __device__ constexpr int direct_prefetch() {
  return DEEP ? (MT == 1 ? 12 : 6) : (NP + MT >= 4 ? 2 : NP + MT == 3 ? 3 : kPrefetchDirect);
}

// SPLIT = false: the caller guarantees KS == 1 (no fixup code, fewer registers).
template <bool BF, int MT, int NP, int NW, bool DEEP, int AM, int EPI, bool COH, bool SPLIT, class Wait>
__device__ bool gemm_tile_direct(const GemmArgs& p, int M, int tile, int split, unsigned char* smem,
                                 float* s_scale, int* s_flag, Wait&& wait) {
  static_assert(MT <= kDirectMT, "direct path row tiles");
  constexpr int P = direct_prefetch<MT, NP, DEEP>();
  constexpr int NTH = NW * 64;
  constexpr int FS = NP * kPairCols + 1;   // row stride of the epilogue tile
  constexpr int QS = MT * NP * 512;        // floats per slice in LDS
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int ns = p.ns, spw = ns / NW;      // slices per split, per wave
  const int kt0 = split * p.ktps;
  const int n_all = min(p.KT, kt0 + p.ktps) - kt0;
  const int s0 = wave * spw;
  const int qa = slice_start(kt0, n_all, s0, ns), n = slice_start(kt0, n_all, s0 + spw, ns) - qa;
  const int pair0 = tile * NP;
  float* R = reinterpret_cast<float*>(smem);   // [slice][mt][pair][j][i][lane]
  float* F = R + ns * QS;

  f4 acc[MT][NP][2];
  auto zero = [&] {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        acc[mt][q][0] = f4{0.f, 0.f, 0.f, 0.f};
        acc[mt][q][1] = f4{0.f, 0.f, 0.f, 0.f};
      }
  };
  zero();
  // slice bookkeeping: slice `sl` of this wave ends after local k-step `next`
  int sl = s0, next = slice_start(kt0, n_all, s0 + 1, ns) - qa;
  auto flush = [&] {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int q = 0; q < NP; ++q)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            R[sl * QS + (((mt * NP + q) * 2 + j) * 4 + i) * 64 + lane] = acc[mt][q][j][i];
    zero();
  };
  // after `done` k-steps: close every slice that has ended (empty ones included)
  auto advance = [&](int done) {
    while (sl < s0 + spw - 1 && next <= done) {
      flush();
      ++sl;
      next = slice_start(kt0, n_all, sl + 1, ns) - qa;
    }
  };

  const uint4* wp = p.W + (size_t)pair0 * p.KT * 128 + lane;
  const size_t pstride = (size_t)p.KT * 128;        // next pair's tiles
  const uint4* ap[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    ap[mt] = static_cast<const uint4*>(p.A) + frag_lane_unit_clamped(lane, M - mt * 16);
  const long long lo = p.a_plane / ET<BF>::PER16;   // lo plane, in 16-byte units
  auto loadW = [&](int kt, uint4(&bb)[NP][2]) {
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      bb[q][0] = ldw(wp + q * pstride + (size_t)kt * 128);
      bb[q][1] = ldw(wp + q * pstride + (size_t)kt * 128 + 64);
    }
  };
  // lanes of rows >= M read row 0 of their tile (frag_lane_unit_clamped):
  // every lane loads, with no branch, so the waits stay exact
  auto loadA = [&](int kt, AFrag(&af)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const uint4* a = ap[mt] + ((size_t)mt * p.KT + kt) * 64;
      af[mt].h = *a;
      if constexpr (BF) af[mt].l = a[lo];
    }
  };
  auto step = [&](int s, const uint4(&bb)[NP][2], const AFrag(&af)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        acc[mt][q][0] = mma_a<BF>(af[mt], bb[q][0], acc[mt][q][0]);
        acc[mt][q][1] = mma_a<BF>(af[mt], bb[q][1], acc[mt][q][1]);
      }
    if (spw > 1) advance(s + 1);
  };
  // Loads retire in issue order, so every k-step's wait is exact only if
  // the loads are always issued in the same order: (W, A) of step s + P
  // right after step s.  The first round is written out apart from the
  // loop because its weights are issued before `wait()` (ahead of the
  // activations); after it the loop is entered with the loads in its own
  // order.  Loads past the end re-read the last k-step (clamped), so no
  // round issues a different number of loads.  A wave whose slices are all
  // empty (splits of fewer k-steps than slices) only joins the wait.
  auto kk = [&](int s) { return qa + min(s, n - 1); };
  uint4 b[P][NP][2];
  AFrag af[P][MT];
#pragma unroll
  for (int u = 0; u < P; ++u)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) af[u][mt] = AFrag{make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
  if (n > 0) {
#pragma unroll
    for (int u = 0; u < P; ++u) loadW(kk(u), b[u]);
  }
  wait();
  constexpr int RPW = (MT * 16 + NW - 1) / NW;   // rows per wave of the row scales
  float rs[RPW];
  row_scale_loads<AM, RPW, NW>(p, M, rs);        // read while the first weights arrive
  if (spw > 1) advance(0);
  if (n > 0) {
#pragma unroll
    for (int u = 0; u < P; ++u) loadA(kk(u), af[u]);
#pragma unroll
    for (int u = 0; u < P; ++u) {
      if (u == 0 || u < n) step(u, b[u], af[u]);
      loadW(kk(u + P), b[u]);
      loadA(kk(u + P), af[u]);
      __builtin_amdgcn_sched_barrier(0);
    }
    int i = P;
    for (; i + P <= n; i += P) {
#pragma unroll
      for (int u = 0; u < P; ++u) {
        step(i + u, b[u], af[u]);
        loadW(kk(i + u + P), b[u]);
        loadA(kk(i + u + P), af[u]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int u = 0; u < P; ++u)
      if (i + u < n) step(i + u, b[u], af[u]);
  }
  // the last slice, then any empty slices after it
  for (;;) {
    flush();
    if (sl >= s0 + spw - 1) break;
    ++sl;
  }

  const bool split_k = SPLIT && p.KS > 1;
  row_scale_finish<AM, RPW, NW>(p, M, rs, s_scale);
  __syncthreads();
  // element x = (((mt * NP + q) * 2 + j) * 4 + i) * 64 + l: row 16 mt + 4 (l / 16) + i,
  // column 32 q + 16 j + l % 16
  auto row_of = [](int x) { return (x >> 6) / (8 * NP) * 16 + 4 * ((x & 63) >> 4) + ((x >> 6) & 3); };
  auto col_of = [](int x) { return ((x >> 9) % NP) * kPairCols + ((x >> 8) & 1) * 16 + (x & 15); };
  auto slice_sum = [&](int x) {
    float v = R[x];
    for (int q = 1; q < ns; ++q) v += R[q * QS + x];
    return v;
  };
  const int n0 = pair0 * kPairCols;
  if (split_k) {
    // split partials through the epilogue tile: F[row][col] first, then publish
    for (int x = tid; x < QS; x += NTH) F[row_of(x) * FS + col_of(x)] = slice_sum(x);
    __syncthreads();
    if (!publish_split<NTH>(p, M, split, n0, NP * kPairCols, &p.counters[tile], s_flag,
                            [&](int m, int c) { return F[m * FS + c]; }))
      return false;
    fixup_rows<AM, NTH>(p, M, n0, NP * kPairCols, 0, M, s_scale, F, FS);
  } else {
    for (int x = tid; x < QS; x += NTH) {
      const int m = row_of(x);
      if (m < M) {
        const float v = slice_sum(x);
        F[m * FS + col_of(x)] = AM == A_NORM ? v * s_scale[m] : v;
      }
    }
  }
  lds_sync();
  epilogue_rows<BF, EPI, COH, NTH>(p, F, FS, pair0, NP, 0, M);
  return true;
}

// Balanced direct path (up to kDirectMT row tiles, one tile pair per unit).
// The units (tile pair, k-split) of a GEMM are numbered pair-major, split
// minor; workgroup b of G takes units [b U / G, (b + 1) U / G), so every
// workgroup streams the same share of the weights (to within one unit)
// whatever the number of pairs, and no compute unit holds more workgroups
// than another.  A unit is summed exactly as gemm_tile_direct sums it with
// kWaves slices per split (wave w: slice w, k-steps in order by MFMA from
// zero; slices added in order in LDS; splits added in order by the fixup),
// so its results are those of the other paths bit for bit.
//   Each wave issues its slices of all the workgroup's units as one run of
// loads, P k-steps ahead across unit boundaries; the barrier that closes a
// unit orders LDS only, so the run stays in flight.  Unit sums collect in
// one LDS tile [row][32 nu + 1]; after the stream come the epilogue of the
// workgroup's pairs (KS = 1), or its split partials and the fixup and
// epilogue of each pair whose last split arrives here.
//   Host-checked: every split has at least kWaves k-steps, at most
// kMaxUnits units per workgroup, G <= U.
//   smem: dynamic LDS of gemm_range_lds_bytes(MT, nu_max); s_flags:
//   kMaxUnits ints.

__host__ __device__ constexpr int gemm_range_lds_bytes(int MT, int nu_max) {
  return (2 * kWaves * MT * 512 + MT * 16 * (nu_max * kPairCols + 1)) * 4;
}

// Launch constants of the balanced path: dynamic LDS of at least
// kRangeMinLds keeps one workgroup per compute unit; kRangePrefetch
// k-steps in flight per wave; slice lengths (KT / kWaves) that have the
// register-resident variant, per element type.
constexpr int kRangeMinLds = 82 * 1024;
constexpr int kRangePrefetch = 4;
template <bool BF> inline constexpr int kRangeSL[3] = {2, 16, 28};
template <> inline constexpr int kRangeSL<false>[3] = {4, 4, 4};

// The balanced path takes the register-resident variant for KS = 1, one
// row tile and a slice length from kRangeSL, for the gate/up and LM-head
// products (normalised A): its slice length, else 0.
template <bool BF>
__host__ __device__ inline int range_ra_slice(int AM, int EPI, int MT, int KS, int KT) {
  if (AM != A_NORM || (EPI != EPI_SWIGLU && EPI != EPI_ARGMAX) || MT != 1 || KS != 1 || KT % kWaves) return 0;
  const int sl = KT / kWaves;
  return sl == kRangeSL<BF>[0] || sl == kRangeSL<BF>[1] || sl == kRangeSL<BF>[2] ? sl : 0;
}

// Closes unit j of the balanced path: this wave's slice sums go to LDS
// slot j & 1, then (all slices present) the slices are added in order into
// columns 32 j .. of F.  Every wave calls it once per unit, in unit order.
template <int MT>
__device__ __forceinline__ void range_close(float* R, float* F, int fs, int j, int wave, f4 (&acc)[MT][2]) {
  constexpr int QS = MT * 512;
  const int tid = threadIdx.x, lane = tid & 63;
  float* Rw = R + ((j & 1) * kWaves + wave) * QS;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
#pragma unroll
      for (int i = 0; i < 4; ++i) Rw[((mt * 2 + jj) * 4 + i) * 64 + lane] = acc[mt][jj][i];
      acc[mt][jj] = f4{0.f, 0.f, 0.f, 0.f};
    }
  lds_sync();
  const float* R0 = R + (j & 1) * kWaves * QS;
  for (int x = tid; x < QS; x += kWaves * 64) {
    float v = R0[x];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) v += R0[q * QS + x];
    // element x = ((mt * 2 + jj) * 4 + i) * 64 + l: row 16 mt + 4 (l / 16) + i, column 16 jj + l % 16
    const int row = (x >> 9) * 16 + 4 * ((x & 63) >> 4) + ((x >> 6) & 3);
    const int col = ((x >> 8) & 1) * 16 + (x & 15);
    F[row * fs + j * kPairCols + col] = v;
  }
}

// After the stream of the balanced path (s_scale already holds the row
// scales): the epilogue of units [u0, u0 + nu) from their sums in F, or,
// with k-splits, their partials and the fixup and epilogue of each pair
// whose last split arrives in this workgroup.
template <bool BF, int AM, int EPI, bool COH>
__device__ __forceinline__ void range_finish(const GemmArgs& p, int M, float* F, int fs, int u0, int nu, const float* s_scale,
                             int* s_flags) {
  constexpr int NTH = kWaves * 64;
  const int tid = threadIdx.x, KS = p.KS;
  const int C = nu * kPairCols;
  if (KS == 1) {
    if constexpr (AM == A_NORM) {
      const int wave = tid >> 6, lane = tid & 63;
      for (int m = wave; m < M; m += kWaves)
        for (int c = lane; c < C; c += 64) F[m * fs + c] *= s_scale[m];
      lds_sync();
    }
    epilogue_rows<BF, EPI, COH, NTH>(p, F, fs, u0, nu, 0, M);
    return;
  }
  for (int e = tid; e < M * C; e += NTH) {
    const int m = e / C, c = e - m * C;
    const int u = u0 + c / kPairCols, pair = u / KS;
    store_partial(&p.part[((size_t)(u - pair * KS) * M + m) * p.N + pair * kPairCols + (c & (kPairCols - 1))],
                  F[m * fs + c]);
  }
  wait_vmem();
  __syncthreads();  // every wave's partial stores are performed
  if (tid < nu) {
    const int pair = (u0 + tid) / KS;
    const bool last = counter_add(&p.counters[pair], 1) == KS - 1;
    if (last) st<true>(&p.counters[pair], 0);  // ready for the next launch
    s_flags[tid] = last;
  }
  __syncthreads();
  for (int j = 0; j < nu; ++j) {
    if (!s_flags[j]) continue;
    const int pair = (u0 + j) / KS;
    fixup_rows<AM, NTH>(p, M, pair * kPairCols, kPairCols, 0, M, s_scale, F + j * kPairCols, fs);
    lds_sync();
    epilogue_rows<BF, EPI, COH, NTH>(p, F + j * kPairCols, fs, pair, 1, 0, M);
    lds_sync();
  }
}

template <bool BF, int MT, int P, int AM, int EPI, bool COH, class Wait>
__device__ __forceinline__ void gemm_range_direct(const GemmArgs& p, int M, unsigned char* smem, float* s_scale, int* s_flags,
                                  Wait&& wait) {
  constexpr int QS = MT * 512;                       // floats of one wave's slice
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KS = p.KS, KT = p.KT, G = p.G;
  const int U = (p.N / kPairCols) * KS;
  const int u0 = (int)((long long)blockIdx.x * U / G), u1 = (int)((long long)(blockIdx.x + 1) * U / G);
  const int nu = u1 - u0;
  const int fs = ((U + G - 1) / G) * kPairCols + 1;
  float* R = reinterpret_cast<float*>(smem);         // [unit & 1][wave][mt][j][i][lane]
  float* F = R + 2 * kWaves * QS;                    // [row][fs]: unit j at columns 32 j ..

  // this wave's k-steps of unit j: slice `wave` of the unit's split
  struct Cur {
    int j, pair, kt, end;
  };
  auto set_unit = [&](Cur& c, int j) {
    const int u = u0 + j;
    c.j = j;
    c.pair = u / KS;
    const int kt0 = (u - c.pair * KS) * p.ktps;
    const int n_all = min(KT, kt0 + p.ktps) - kt0;
    c.kt = slice_start(kt0, n_all, wave, kWaves);
    c.end = slice_start(kt0, n_all, wave + 1, kWaves);
  };
  int S = 0;                                          // k-steps of this wave
  for (int j = 0; j < nu; ++j) {
    Cur c;
    set_unit(c, j);
    S += c.end - c.kt;
  }

  const uint4* ap[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    ap[mt] = static_cast<const uint4*>(p.A) + frag_lane_unit_clamped(lane, M - mt * 16);
  const long long lo = p.a_plane / ET<BF>::PER16;   // lo plane, in 16-byte units
  // one k-step: the pair's two weight tiles, then the row tiles' fragments
  // (lanes of rows >= M read row 0 of their tile: no branch, exact waits)
  auto loadW = [&](const Cur& c, uint4(&bb)[2]) {
    const uint4* w = p.W + ((size_t)c.pair * KT + c.kt) * 128 + lane;
    bb[0] = ldw(w);
    bb[1] = ldw(w + 64);
  };
  auto loadA = [&](const Cur& c, AFrag(&af)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const uint4* a = ap[mt] + ((size_t)mt * KT + c.kt) * 64;
      af[mt].h = ldg(a);
      if constexpr (BF) af[mt].l = ldg(a + lo);
    }
  };
  auto load = [&](const Cur& c, uint4(&bb)[2], AFrag(&af)[MT]) {
    loadW(c, bb);
    loadA(c, af);
  };
  // the load cursor steps through the units; past the last k-step it
  // re-reads that k-step, so every round issues the same loads
  auto advance = [&](Cur& c) {
    if (++c.kt == c.end) {
      if (c.j + 1 < nu) set_unit(c, c.j + 1);
      else c.kt = c.end - 1;
    }
  };

  f4 acc[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt][0] = acc[mt][1] = f4{0.f, 0.f, 0.f, 0.f};
  uint4 bw[P][2];
  AFrag af[P][MT];
#pragma unroll
  for (int u = 0; u < P; ++u)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) af[u][mt] = AFrag{make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
  Cur cl;
  set_unit(cl, 0);
  int rem = cl.end - cl.kt;                           // k-steps left in the unit being summed
  // the first round: weights first, then (after `wait()`, which the
  // persistent kernel uses to wait for the producer of A) the activations
  {
    Cur ca = cl;
#pragma unroll
    for (int u = 0; u < P; ++u) {
      loadW(cl, bw[u]);
      advance(cl);
    }
    wait();
#pragma unroll
    for (int u = 0; u < P; ++u) {
      loadA(ca, af[u]);
      advance(ca);
    }
  }
  constexpr int RPW = MT * 16 / kWaves;
  float rs[RPW];
  row_scale_loads<AM, RPW>(p, M, rs);                 // read while the first weights arrive
  int cj = 0;                                         // unit being summed
  for (int i = 0; i < S; i += P) {
#pragma unroll
    for (int u = 0; u < P; ++u) {
      if (i + u < S) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          acc[mt][0] = mma_a<BF>(af[u][mt], bw[u][0], acc[mt][0]);
          acc[mt][1] = mma_a<BF>(af[u][mt], bw[u][1], acc[mt][1]);
        }
        if (--rem == 0) {
          range_close<MT>(R, F, fs, cj, wave, acc);
          if (++cj < nu) {
            Cur c;
            set_unit(c, cj);
            rem = c.end - c.kt;
          }
        }
      }
      load(cl, bw[u], af[u]);
      advance(cl);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  row_scale_finish<AM, RPW>(p, M, rs, s_scale);
  lds_sync();                                         // the last unit's sums are in F
  range_finish<BF, AM, EPI, COH>(p, M, F, fs, u0, nu, s_scale, s_flags);
}

// The balanced path for KS = 1 and one row tile when every wave's slice
// has SL = KT / kWaves k-steps: a wave's slice covers the same k-steps of
// every pair, so its activation fragments are loaded once into registers
// and only the weights stream.  Sums as in gemm_range_direct.
template <bool BF, int P, int SL, int AM, int EPI, bool COH, class Wait>
__device__ __forceinline__ void gemm_range_direct_ra(const GemmArgs& p, int M, unsigned char* smem, float* s_scale, int* s_flags,
                                     Wait&& wait) {
  static_assert(SL % P == 0, "slice length must be a multiple of the prefetch depth");
  constexpr int QS = 512;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KT = p.KT, G = p.G;
  const int U = p.N / kPairCols;
  const int u0 = (int)((long long)blockIdx.x * U / G), u1 = (int)((long long)(blockIdx.x + 1) * U / G);
  const int nu = u1 - u0;
  const int fs = ((U + G - 1) / G) * kPairCols + 1;
  float* R = reinterpret_cast<float*>(smem);
  float* F = R + 2 * kWaves * QS;
  const int kt0 = wave * SL;                          // slice_start(0, KT, wave, kWaves)
  const uint4* wb = p.W + ((size_t)u0 * KT + kt0) * 128 + lane;
  // weights of k-step s of unit j; past the last unit, its last k-step again
  auto loadW = [&](int j, int s, uint4(&bb)[2]) {
    const bool past = j >= nu;
    const uint4* w = wb + ((size_t)(past ? nu - 1 : j) * KT + (past ? SL - 1 : s)) * 128;
    bb[0] = ldw(w);
    bb[1] = ldw(w + 64);
  };
  uint4 bw[P][2];
#pragma unroll
  for (int u = 0; u < P; ++u) loadW(0, u, bw[u]);
  wait();   // the persistent kernel waits here for the producer of A
  const uint4* ap = static_cast<const uint4*>(p.A) + frag_lane_unit_clamped(lane, M) + (size_t)kt0 * 64;
  const long long lo = p.a_plane / ET<BF>::PER16;
  AFrag af[SL];
#pragma unroll
  for (int s = 0; s < SL; ++s) {
    af[s].h = ldg(ap + (size_t)s * 64);
    if constexpr (BF) af[s].l = ldg(ap + (size_t)s * 64 + lo);
  }
  float rs[16 / kWaves];
  row_scale_loads<AM, 16 / kWaves>(p, M, rs);
  f4 acc[1][2];
  acc[0][0] = acc[0][1] = f4{0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < nu; ++j) {
#pragma unroll
    for (int s = 0; s < SL; ++s) {
      acc[0][0] = mma_a<BF>(af[s], bw[s % P][0], acc[0][0]);
      acc[0][1] = mma_a<BF>(af[s], bw[s % P][1], acc[0][1]);
      loadW(j + (s + P) / SL, (s + P) % SL, bw[s % P]);
      __builtin_amdgcn_sched_barrier(0);
    }
    range_close<1>(R, F, fs, j, wave, acc);
  }
  row_scale_finish<AM, 16 / kWaves>(p, M, rs, s_scale);
  lds_sync();
  range_finish<BF, AM, EPI, COH>(p, M, F, fs, u0, nu, s_scale, s_flags);
}

// Staged path (more than kDirectMT row tiles): a workgroup owns kPairsS NPW
// tile pairs (NPW per wave) of one split, for row tiles [mt0, mt0 + MT);
// each wave keeps its slices apart in registers (running sum S).  The
// split's slices are cut into chunks of at most CK k-steps; a chunk's
// activation fragments are staged in LDS and shared by the waves, its
// weights held in registers.  Two LDS buffers: the next chunk's weights
// and activation fragments are requested before the current chunk is
// summed and written to the other buffer after it, so memory latency
// overlaps the MFMA work.  Row groups (mt0 > 0) let narrow matrices use
// more workgroups; `cnt` is the split counter of this (pairs, rows) tile
// (default: the pair group).
// WC: weight tiles by ordinary cached loads (the other row groups of the
// pass read them again from L2), else by streaming loads.
//   smem: dynamic LDS of gemm_staged_lds_bytes<BF, MT, NPW>().

template <bool BF, int MT> __host__ __device__ constexpr int staged_ck() {
  constexpr int per = 2 * (BF ? 2 : 1) * MT * 1024;   // both buffers, one k-step
  constexpr int cap = MT == 2 || MT == 3 ? 2 : 4;     // row groups of 2-3 tiles: few enough registers for 4 workgroups per CU
  return kStagedLds / per > cap ? cap : kStagedLds / per;
}
// Epilogue tile of the staged path with NPW pairs per wave: row stride
// (floats) and rows per pass (at most the workgroup's rows).
template <int NPW> __host__ __device__ constexpr int staged_fstride() { return kPairsS * NPW * kPairCols + 4; }
template <int MT> __host__ __device__ constexpr int staged_frows() { return MT * 16 < kFRows ? MT * 16 : kFRows; }
template <bool BF, int MT, int NPW = 1> __host__ __device__ constexpr int gemm_staged_lds_bytes() {
  constexpr int a = 2 * (BF ? 2 : 1) * MT * staged_ck<BF, MT>() * 1024;
  constexpr int f = staged_frows<MT>() * staged_fstride<NPW>() * 4;
  return a > f ? a : f;
}

template <bool BF, int MT, int AM, int EPI, bool COH, bool WC = false, int NPW = 1>
__device__ bool gemm_tile_staged(const GemmArgs& p, int M, int group, int split, unsigned char* smem,
                                 float* s_scale, int* s_flag, int mt0 = 0, int cnt = -1) {
  constexpr int kRegions = BF ? 2 : 1;
  constexpr int PG = kPairsS * NPW;                // pairs of the workgroup, NPW per wave
  constexpr int CK = staged_ck<BF, MT>();
  constexpr int BUF = kRegions * MT * CK * 64;     // 16-byte elements per buffer
  constexpr int NV = (BUF + 255) / 256;            // of which each thread stages at most NV
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kt0 = split * p.ktps;
  const int n_all = min(p.KT, kt0 + p.ktps) - kt0;
  const size_t pstride = (size_t)p.KT * 128;                                   // 16-byte units per pair
  const uint4* wp = p.W + (size_t)(group * PG + wave * NPW) * pstride + lane;   // this wave's first pair
  const uint4* ag = static_cast<const uint4*>(p.A);
  const long long lo = p.a_plane / ET<BF>::PER16;
  uint4* la = reinterpret_cast<uint4*>(smem);     // [buffer][region][mt][k-step of chunk][lane]

  // chunk (slice q, first k-step c0, n k-steps); q == ns: past the end
  struct Chunk {
    int q, c0, n;
  };
  auto first_of = [&](int q) {
    Chunk c;
    c.q = q;
    c.c0 = slice_start(kt0, n_all, q, p.ns);
    c.n = min(slice_start(kt0, n_all, q + 1, p.ns) - c.c0, CK);
    return c;
  };
  auto next_of = [&](const Chunk& c) {
    const int qb = slice_start(kt0, n_all, c.q + 1, p.ns);
    if (c.c0 + c.n < qb) {
      Chunk d = c;
      d.c0 += c.n;
      d.n = min(qb - d.c0, CK);
      return d;
    }
    return first_of(c.q + 1);
  };
  // element u of chunk d's staging: block (region, tile, k-step) u / 64,
  // position u % 64 of the block in LDS, which holds the 16-byte unit lane
  // u % 64 feeds to the MFMA (frag_lane_unit): the waves then read their
  // fragments as 64 consecutive units, free of bank conflicts (read in
  // fragment order, lanes 64 bytes apart, four of eight lanes met in one
  // bank); returns its source and sets its place in a buffer.  A tile past
  // the pass's last one (the last row group of a pass may reach beyond
  // kMaxMTiles) loads the last one instead: its rows are never stored.
  const int mt_last = (M - 1) >> 4;
  auto elem = [&](const Chunk& d, int u, int& dst) {
    const int pos = u & 63, b = u >> 6;
    const int rg = b / (MT * d.n), r2 = b - rg * (MT * d.n);
    const int mt = r2 / d.n, r = r2 - mt * d.n;
    dst = ((rg * MT + mt) * CK + r) * 64 + pos;
    return ag + rg * lo + ((size_t)min(mt0 + mt, mt_last) * p.KT + d.c0 + r) * 64 + frag_lane_unit(pos);
  };
  // requests chunk d: CK k-steps of weights (past the chunk its last
  // again, clamped to the matrix: unused) and this thread's NV staging
  // elements (u = tid + 256 i; past the chunk's last element that one
  // again: no branch around the loads, so they all stay in flight)
  auto request = [&](const Chunk& d, uint4(&wb)[CK][NPW][2], uint4(&av)[NV], int(&ad)[NV]) {
#pragma unroll
    for (int r = 0; r < CK; ++r) {
      const size_t kp = (size_t)min(d.c0 + min(r, max(d.n, 1) - 1), p.KT - 1) * 128;
#pragma unroll
      for (int q = 0; q < NPW; ++q) {
        if constexpr (WC) {
          wb[r][q][0] = ldg(wp + q * pstride + kp);
          wb[r][q][1] = ldg(wp + q * pstride + kp + 64);
        } else {
          wb[r][q][0] = ldw(wp + q * pstride + kp);
          wb[r][q][1] = ldw(wp + q * pstride + kp + 64);
        }
      }
    }
    const int total = max(kRegions * MT * d.n * 64, 1);
#pragma unroll
    for (int i = 0; i < NV; ++i) av[i] = ldg(elem(d, min((int)tid + 256 * i, total - 1), ad[i]));
  };
  auto stage = [&](const Chunk& d, uint4* buf, const uint4(&av)[NV], const int(&ad)[NV]) {
    const int total = kRegions * MT * d.n * 64;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if ((int)tid + 256 * i < total) buf[ad[i]] = av[i];
  };

  f4 S[MT][NPW][2], acc[MT][NPW][2];
  uint4 w0[CK][NPW][2], w1[CK][NPW][2], av[NV];
  int ad[NV];
  // one chunk: request the next one (weights into wn, fragments into
  // registers), sum this one from LDS buffer bi with weights wc, stage the
  // next one into the other buffer; false after the last chunk
  auto step = [&](Chunk& cur, int bi, const uint4(&wc)[CK][NPW][2], uint4(&wn)[CK][NPW][2]) {
    const Chunk nxt = next_of(cur);
    const bool more = nxt.q < p.ns;
    // after the last chunk, the current one again (unused): the same loads
    // on every path keep the compiler's waits exact
    request(more ? nxt : cur, wn, av, ad);
    if (cur.c0 == slice_start(kt0, n_all, cur.q, p.ns)) {   // a slice begins
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int q = 0; q < NPW; ++q) {
          acc[mt][q][0] = f4{0.f, 0.f, 0.f, 0.f};
          acc[mt][q][1] = f4{0.f, 0.f, 0.f, 0.f};
        }
    }
    const uint4* lb = la + bi * BUF;
#pragma unroll
    for (int ks = 0; ks < CK; ++ks) {
      if (ks < cur.n) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          AFrag af;
          af.h = lb[(mt * CK + ks) * 64 + lane];
          if constexpr (BF) af.l = lb[MT * CK * 64 + (mt * CK + ks) * 64 + lane];
#pragma unroll
          for (int q = 0; q < NPW; ++q) {
            acc[mt][q][0] = mma_a<BF>(af, wc[ks][q][0], acc[mt][q][0]);
            acc[mt][q][1] = mma_a<BF>(af, wc[ks][q][1], acc[mt][q][1]);
          }
        }
      }
    }
    if (cur.c0 + cur.n == slice_start(kt0, n_all, cur.q + 1, p.ns)) {   // the slice ends
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int q = 0; q < NPW; ++q)
#pragma unroll
          for (int j = 0; j < 2; ++j) S[mt][q][j] = cur.q == 0 ? acc[mt][q][j] : S[mt][q][j] + acc[mt][q][j];
    }
    if (!more) return false;
    // the other buffer was last read in the previous chunk, before the
    // barrier that ended it
    stage(nxt, la + (bi ^ 1) * BUF, av, ad);
    lds_sync();
    cur = nxt;
    return true;
  };
  Chunk cur = first_of(0);
  request(cur, w0, av, ad);
  stage(cur, la, av, ad);
  lds_sync();
  // chunks alternate between buffers 0 and 1 and weight sets w0 and w1
  while (step(cur, 0, w0, w1) && step(cur, 1, w1, w0)) {
  }
  lds_sync();   // the A buffers are no longer read (F reuses the LDS)

  float* F = reinterpret_cast<float*>(smem);
  constexpr int FS = staged_fstride<NPW>(), FR = staged_frows<MT>();
  const int n0 = group * PG * kPairCols, C = PG * kPairCols;
  const int R0 = mt0 * 16, R1 = min(M, (mt0 + MT) * 16);   // this workgroup's rows
  if (cnt < 0) cnt = group;
  // lane's value of (row m, column 32 (NPW wave + q) + 16 j + lane % 16)
  auto put = [&](int r0, int r1, bool scale) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int q = 0; q < NPW; ++q)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = (mt0 + mt) * 16 + (lane >> 4) * 4 + i;
            const int col = (wave * NPW + q) * kPairCols + j * 16 + (lane & 15);
            if (row >= r0 && row < r1)
              F[(row - r0) * FS + col] = AM == A_NORM && scale ? S[mt][q][j][i] * s_scale[row] : S[mt][q][j][i];
          }
  };
  if (p.KS > 1) {
    // publish in row blocks through F
    for (int r0 = R0; r0 < R1; r0 += FR) {
      const int r1 = min(R1, r0 + FR);
      lds_sync();
      put(r0, r1, false);
      __syncthreads();
      for (int e = tid; e < (r1 - r0) * C; e += 256) {
        const int m = r0 + e / C, c = e % C;
        store_partial(&p.part[((size_t)split * M + m) * p.N + n0 + c], F[(m - r0) * FS + c]);
      }
    }
    wait_vmem();
    __syncthreads();
    if (tid == 0) *s_flag = counter_add(&p.counters[cnt], 1) == p.KS - 1;
    __syncthreads();
    if (!*s_flag) return false;
    if (tid == 0) st<true>(&p.counters[cnt], 0);
    row_scales<AM>(p, M, s_scale);
    __syncthreads();
    for (int r0 = R0; r0 < R1; r0 += FR) {
      const int r1 = min(R1, r0 + FR);
      fixup_rows<AM>(p, M, n0, C, r0, r1, s_scale, F, FS);
      lds_sync();
      epilogue_rows<BF, EPI, COH>(p, F, FS, group * PG, PG, r0, r1);
      lds_sync();
    }
  } else {
    row_scales<AM>(p, M, s_scale);
    __syncthreads();  // A tiles no longer read; s_scale written
    for (int r0 = R0; r0 < R1; r0 += FR) {
      const int r1 = min(R1, r0 + FR);
      put(r0, r1, true);
      lds_sync();
      epilogue_rows<BF, EPI, COH>(p, F, FS, group * PG, PG, r0, r1);
      lds_sync();
    }
  }
  return true;
}

// ---------------------------------------------------------------------------
// Arg-max of row `row` over the LM head's per-pair partials (256 threads):
// larger value wins, equal values keep the lower token id; *bad is set for a
// non-finite logit and *margin receives the gap between the largest and
// the second-largest logit of the row (0 when two token ids tie).  The
// (value, id, second) partials merge as: the winner's value and id, and
// the larger of the loser's value and the winner's second; the winner is
// decided by the total order (value descending, id ascending), so the
// result does not depend on the order of the merges.  s4f, s4s / s4i:
// 4-entry LDS scratch.

__device__ __forceinline__ void top2_merge(float& v, int& i, float& v2, float ov, int oi, float ov2) {
  if (ov > v || (ov == v && oi < i)) {
    v2 = fmaxf(v, ov2);
    v = ov;
    i = oi;
  } else {
    v2 = fmaxf(v2, ov);
  }
}

template <bool COH>
__device__ __forceinline__ void argmax_row(const float* amax_val, const float* amax_val2, const int* amax_idx,
                                           int n_pairs, int row, int* tok, int* bad, float* margin, float* s4f,
                                           float* s4s, int* s4i) {
  constexpr int kPer = 8;   // pairs per thread, loads in flight together
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  float best = -INFINITY, second = -INFINITY;
  int bi = 0x7fffffff;
  bool b = false;
  auto ld = [](const auto* q) { if constexpr (COH) return ld_coherent(q); else return *q; };
  for (int g0 = 0; g0 < n_pairs; g0 += 256 * kPer) {
    float v[kPer], v2[kPer];
    int id[kPer];
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int g = g0 + t * 256 + tid;
      if (g < n_pairs) {
        v[t] = ld(amax_val + (size_t)row * n_pairs + g);
        v2[t] = ld(amax_val2 + (size_t)row * n_pairs + g);
        id[t] = ld(amax_idx + (size_t)row * n_pairs + g);
      }
    }
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int g = g0 + t * 256 + tid;
      if (g < n_pairs) {
        if (!isfinite(v[t])) b = true;
        else top2_merge(best, bi, second, v[t], id[t], v2[t]);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(best, o), ov2 = __shfl_xor(second, o);
    const int oi = __shfl_xor(bi, o);
    top2_merge(best, bi, second, ov, oi, ov2);
  }
  const bool wb = __ballot(b) != 0;
  if (lane == 0) { s4f[wave] = best; s4s[wave] = second; s4i[wave] = bi | (wb ? 0x80000000 : 0); }
  __syncthreads();
  if (tid == 0) {
    float bv = s4f[0], bv2 = s4s[0];
    int bx = s4i[0] & 0x7fffffff, bb = s4i[0] < 0;
    for (int w = 1; w < 4; ++w) {
      top2_merge(bv, bx, bv2, s4f[w], s4i[w] & 0x7fffffff, s4s[w]);
      bb |= s4i[w] < 0;
    }
    *tok = bx;
    *bad = bb | !isfinite(bv);
    *margin = bv - bv2;
  }
  __syncthreads();
}

// Greedy verification of one request from its rows' greedy tokens
// (Section 4.2; Appendix C.2): accepted = first row i < W-1 whose greedy
// token differs from its candidate (W-1 if none); the correction is the
// greedy token of row `accepted`.
template <class TokAt>
__device__ __forceinline__ StepOut verify_request(const RowDesc* rows, const ReqDesc& rq, TokAt&& tok_at, int bad) {
  int a = 0;
  while (a < rq.W - 1 && rows[rq.row_start + a].cmp == tok_at(rq.row_start + a)) ++a;
  return StepOut{a, tok_at(rq.row_start + a), bad, 0};
}

}  // namespace as2d
