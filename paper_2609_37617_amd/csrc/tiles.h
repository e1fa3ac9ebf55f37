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
// and per-row sum-of-squares partials over 128-column groups.  256 threads;
// srow: LDS scratch of H floats.

template <bool BF, bool COH>
__device__ void embed_row(const RowDesc* __restrict__ rows, int m, const typename ET<BF>::T* __restrict__ embed,
                          const typename ET<BF>::T* __restrict__ audio, int H, const float* __restrict__ gain,
                          float* __restrict__ x, float* __restrict__ sumsq, void* __restrict__ xg,
                          long long xg_plane, float* srow) {
  using T = typename ET<BF>::T;
  constexpr int kPer = 8, kPasses = 4;   // H <= 256 * 8 * 4
  const RowDesc rd = rows[m];
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
        store_act<BF, COH>(xg, xg_plane, (size_t)m * H + c0 + t, v[ps][t] * gain[c0 + t]);
        srow[c0 + t] = v[ps][t];
      }
    }
  }
  lds_sync();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int g = wave; g < H / 128; g += 4) {
    const float v0 = srow[g * 128 + lane], v1 = srow[g * 128 + 64 + lane];
    const float s = wave_sum(v0 * v0 + v1 * v1);
    if (lane == 0) st<COH>(sumsq + g * kMaxRows + m, s);
  }
}

// ---------------------------------------------------------------------------
// Fused GEMM epilogues over rows [r0, r1) of one 128-column group; F holds
// the group's finished values (float32, row stride kFStride).

template <bool BF, int EPI, bool COH>
__device__ void epilogue_rows(const GemmArgs& p, float* F, int group, int r0, int r1) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int N = p.N;
  if constexpr (EPI == EPI_RESID) {
    // x_out = x + Y; planes of x_out * g for the next RMSNorm; sum of squares
    for (int idx = tid; idx < (r1 - r0) * 128; idx += 256) {
      const int m = r0 + (idx >> 7), c = idx & 127;
      const int n = group * 128 + c;
      const size_t o = (size_t)m * N + n;
      const float v = p.x[o] + F[(m - r0) * kFStride + c];
      st<COH>(p.x_out + o, v);
      store_act<BF, COH>(p.out, p.out_plane, o, v * p.gain_next[n]);
      F[(m - r0) * kFStride + c] = v;
    }
    lds_sync();
    for (int m = r0 + wave; m < r1; m += 4) {
      const float v0 = F[(m - r0) * kFStride + lane], v1 = F[(m - r0) * kFStride + 64 + lane];
      const float s = wave_sum(v0 * v0 + v1 * v1);
      if (lane == 0) st<COH>(p.sumsq_out + group * kMaxRows + m, s);
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int F2 = N / 2;
    for (int idx = tid; idx < (r1 - r0) * 64; idx += 256) {
      const int m = r0 + (idx >> 6), c = idx & 63;
      const float g = F[(m - r0) * kFStride + c], u = F[(m - r0) * kFStride + 64 + c];
      store_act<BF, COH>(p.out, p.out_plane, (size_t)m * F2 + group * 64 + c, g / (1.0f + expf(-g)) * u);
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int d = p.head_dim, half = d >> 1;
    const int q_cols = p.n_q * d, qk_cols = (p.n_q + p.n_kv) * d;
    for (int idx = tid; idx < (r1 - r0) * 128; idx += 256) {
      const int m = r0 + (idx >> 7), c = idx & 127;
      const int n = group * 128 + c;
      const RowDesc rd = p.rows[m];
      const float* Fr = F + (m - r0) * kFStride;
      float v = Fr[c] + (p.bias ? p.bias[n] : 0.0f);
      const int dd = n % d;
      if (n < qk_cols) {
        const int i = dd % half;
        const int pc = dd < half ? c + half : c - half;
        const int pn = dd < half ? n + half : n - half;
        const float partner = Fr[pc] + (p.bias ? p.bias[pn] : 0.0f);
        const float cs = p.rope_cs[((size_t)rd.pos * half + i) * 2];
        const float sn = p.rope_cs[((size_t)rd.pos * half + i) * 2 + 1];
        v = dd < half ? v * cs - partner * sn : v * cs + partner * sn;
        if (n < q_cols) {
          st<COH>(p.q_out + (size_t)m * q_cols + n, v);
        } else {
          const int kvh = (n - q_cols) / d;
          st<COH>(p.k_cache + (size_t)rd.slot * p.slot_stride + ((size_t)kvh * p.kv_cap + rd.pos) * d + dd, v);
        }
      } else {
        const int kvh = (n - qk_cols) / d;
        st<COH>(p.v_cache + (size_t)rd.slot * p.slot_stride + ((size_t)kvh * p.kv_cap + rd.pos) * d + dd, v);
      }
    }
  } else {  // EPI_ARGMAX
    for (int m = r0 + wave; m < r1; m += 4) {
      const float v0 = F[(m - r0) * kFStride + lane], v1 = F[(m - r0) * kFStride + 64 + lane];
      const int n0 = group * 128 + lane;
      if (p.logits) {
        p.logits[(size_t)m * N + n0] = v0;   // read by the host only
        p.logits[(size_t)m * N + n0 + 64] = v1;
      }
      const bool bad = !(isfinite(v0) && isfinite(v1));
      float best = v0;
      int bi = n0;
      if (v1 > best) { best = v1; bi = n0 + 64; }
      wave_argmax(best, bi);
      const bool any_bad = __ballot(bad) != 0;
      if (lane == 0) {
        st<COH>(p.amax_val + group * kMaxRows + m, any_bad ? __builtin_nanf("") : best);
        st<COH>(p.amax_idx + group * kMaxRows + m, bi);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// One GEMM tile: 128-column group `group`, k-split `split` (see
// kernels.hip for the scheme).  256 threads.  `wait()` is called after the
// first weight loads are issued and before any activation is read (the
// persistent kernel waits there for the producer of A).  Returns true when
// this workgroup finished the group (ran its epilogue).
//   smem: dynamic LDS (A staging for MT > kDirectMT, then the epilogue
//   tile); s_scale: kMaxRows floats; s_flag: one int.

template <bool BF, int MT, int AM, int EPI, bool COH, class Wait>
__device__ bool gemm_tile(const GemmArgs& p, int M, int group, int split, unsigned char* smem, float* s_scale,
                          int* s_flag, int chunk_kt, Wait&& wait) {
  using T = typename ET<BF>::T;
  constexpr int PER16 = ET<BF>::PER16;
  constexpr int KE = 4 * PER16;           // elements per k-step
  constexpr bool kDirect = MT <= kDirectMT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kt0 = split * p.ktps;
  const int kt1 = min(p.KT, kt0 + p.ktps);
  const int K = p.K;

  f4 acc[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt][0] = f4{0.f, 0.f, 0.f, 0.f};
    acc[mt][1] = f4{0.f, 0.f, 0.f, 0.f};
  }
  const uint4* wp = p.W + (size_t)(group * kWaves + wave) * p.KT * 128 + lane;
  auto step = [&](const uint4(&bb)[2], const AFrag(&af)[MT]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      acc[mt][0] = mma_a<BF>(af[mt], bb[0], acc[mt][0]);
      acc[mt][1] = mma_a<BF>(af[mt], bb[1], acc[mt][1]);
    }
  };

  if constexpr (kDirect) {
    // A fragments straight from the activation planes (rows >= M read
    // values that only reach output rows that are never stored)
    const T* abase = (const T*)p.A + (size_t)(lane & 15) * K + (lane >> 4) * PER16;
    auto loadW = [&](int kt, uint4(&bb)[2]) {
      bb[0] = ldw(wp + (size_t)kt * 128);
      bb[1] = ldw(wp + (size_t)kt * 128 + 64);
    };
    auto loadA = [&](int kt, AFrag(&af)[MT]) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const T* a = abase + (size_t)mt * 16 * K + (size_t)kt * KE;
        af[mt].h = *reinterpret_cast<const uint4*>(a);
        if constexpr (BF) af[mt].l = *reinterpret_cast<const uint4*>(a + p.a_plane);
      }
    };
    const int n = kt1 - kt0;
    uint4 b[kPrefetch][2];
    AFrag af[kPrefetch][MT];
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) loadW(kt0 + min(u, n - 1), b[u]);
    wait();
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) loadA(kt0 + min(u, n - 1), af[u]);
    int i = 0;
    for (; i + 2 * kPrefetch <= n; i += kPrefetch) {
#pragma unroll
      for (int u = 0; u < kPrefetch; ++u) {
        step(b[u], af[u]);
        loadW(kt0 + i + u + kPrefetch, b[u]);
        loadA(kt0 + i + u + kPrefetch, af[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      if (i + u < n) {
        step(b[u], af[u]);
        if (i + u + kPrefetch < n) {
          loadW(kt0 + i + u + kPrefetch, b[u]);
          loadA(kt0 + i + u + kPrefetch, af[u]);
        }
      }
    }
    i += kPrefetch;
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u)
      if (i + u < n) step(b[u], af[u]);
  } else {
    // stage the A planes of `chunk_kt` k-steps in LDS (hi region, then lo)
    wait();
    constexpr int kRegions = BF ? 2 : 1;
    const int stride = lds_row_stride(chunk_kt);
    const int region = MT * 16 * stride;
    const unsigned char* lbase = smem + (lane & 15) * stride + (lane >> 4) * 16;
    for (int c0 = kt0; c0 < kt1; c0 += chunk_kt) {
      const int c1 = min(kt1, c0 + chunk_kt);
      const int n = c1 - c0;
      if (c0 != kt0) lds_sync();
      const int units = kRegions * MT * 16 * n * 4;
      for (int u = tid; u < units; u += 256) {
        const int rg = u / (MT * 16 * n * 4);
        const int r2 = u - rg * (MT * 16 * n * 4);
        const int m = r2 / (n * 4), r = r2 - m * (n * 4);
        const size_t e = (size_t)m * K + (size_t)(c0 + (r >> 2)) * KE + (r & 3) * PER16 + rg * p.a_plane;
        *reinterpret_cast<uint4*>(smem + rg * region + m * stride + (r >> 2) * 64 + (r & 3) * 16) =
            *reinterpret_cast<const uint4*>((const T*)p.A + e);
      }
      uint4 b[kPrefetch][2];
#pragma unroll
      for (int u = 0; u < kPrefetch; ++u) {
        const size_t kp = (size_t)(c0 + min(u, n - 1)) * 128;
        b[u][0] = ldw(wp + kp);
        b[u][1] = ldw(wp + kp + 64);
      }
      lds_sync();
      auto lds_a = [&](int ks, AFrag(&af)[MT]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          af[mt].h = *reinterpret_cast<const uint4*>(lbase + mt * 16 * stride + ks * 64);
          if constexpr (BF) af[mt].l = *reinterpret_cast<const uint4*>(lbase + region + mt * 16 * stride + ks * 64);
        }
      };
      int i = 0;
      for (; i + 2 * kPrefetch <= n; i += kPrefetch) {
#pragma unroll
        for (int u = 0; u < kPrefetch; ++u) {
          AFrag af[MT];
          lds_a(i + u, af);
          step(b[u], af);
          const size_t kn = (size_t)(c0 + i + u + kPrefetch) * 128;
          b[u][0] = ldw(wp + kn);
          b[u][1] = ldw(wp + kn + 64);
        }
      }
#pragma unroll
      for (int u = 0; u < kPrefetch; ++u) {
        if (i + u < n) {
          AFrag af[MT];
          lds_a(i + u, af);
          step(b[u], af);
          if (i + u + kPrefetch < n) {
            const size_t kn = (size_t)(c0 + i + u + kPrefetch) * 128;
            b[u][0] = ldw(wp + kn);
            b[u][1] = ldw(wp + kn + 64);
          }
        }
      }
      i += kPrefetch;
#pragma unroll
      for (int u = 0; u < kPrefetch; ++u) {
        if (i + u < n) {
          AFrag af[MT];
          lds_a(i + u, af);
          step(b[u], af);
        }
      }
    }
  }

  if constexpr (AM == A_NORM) {
    for (int m = tid; m < M; m += 256) {
      float ss = 0.0f;
      for (int g = 0; g < p.n_norm_groups; ++g) ss += p.sumsq[g * kMaxRows + m];
      s_scale[m] = 1.0f / sqrtf(ss / (float)K + p.eps);
    }
  }
  float* F = reinterpret_cast<float*>(smem);
  if (p.KS > 1) {
    // publish this split's partial, then let the last split of the group reduce
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = mt * 16 + (lane >> 4) * 4 + i;
          const int col = group * 128 + (wave * 2 + j) * 16 + (lane & 15);
          if (row < M) store_partial(&p.part[((size_t)split * M + row) * p.N + col], acc[mt][j][i]);
        }
    wait_vmem();
    __syncthreads();  // every wave's partial stores are performed
    if (tid == 0) *s_flag = counter_add(&p.counters[group], 1) == p.KS - 1;
    __syncthreads();
    if (!*s_flag) return false;
    if (tid == 0) st<true>(&p.counters[group], 0);  // ready for the next launch
    for (int r0 = 0; r0 < M; r0 += kFRows) {
      const int r1 = min(M, r0 + kFRows);
      // each element is summed in split order, its split loads issued together
      for (int idx = tid; idx < (r1 - r0) * 128; idx += 256) {
        const int m = r0 + (idx >> 7), c = idx & 127;
        constexpr int kB = 16;
        float sum = 0.0f;
        for (int s0 = 0; s0 < p.KS; s0 += kB) {
          float v[kB];
#pragma unroll
          for (int b = 0; b < kB; ++b)
            if (s0 + b < p.KS) v[b] = load_partial(&p.part[((size_t)(s0 + b) * M + m) * p.N + group * 128 + c]);
#pragma unroll
          for (int b = 0; b < kB; ++b)
            if (s0 + b < p.KS) sum += v[b];
        }
        F[(m - r0) * kFStride + c] = AM == A_NORM ? sum * s_scale[m] : sum;
      }
      lds_sync();
      epilogue_rows<BF, EPI, COH>(p, F, group, r0, r1);
      lds_sync();
    }
  } else {
    __syncthreads();  // A tiles no longer read; s_scale written
    for (int r0 = 0; r0 < M; r0 += kFRows) {
      const int r1 = min(M, r0 + kFRows);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = mt * 16 + (lane >> 4) * 4 + i;
            const int col = (wave * 2 + j) * 16 + (lane & 15);
            if (row >= r0 && row < r1)
              F[(row - r0) * kFStride + col] = AM == A_NORM ? acc[mt][j][i] * s_scale[row] : acc[mt][j][i];
          }
      lds_sync();
      epilogue_rows<BF, EPI, COH>(p, F, group, r0, r1);
      lds_sync();
    }
  }
  return true;
}

// ---------------------------------------------------------------------------
// Attention over one 32-key chunk c of request r for query head h (see
// kernels.hip).  256 threads; smem: dynamic LDS of attn_lds_bytes(D).

template <int D> __host__ __device__ constexpr int attn_lds_bytes() {
  return (2 * kAttnChunk * (D + 1) + 4 * D + 4 * kAttnChunk) * 4;
}

template <int D, bool COH>
__device__ void attn_chunk_tile(const AttnArgs& p, int c, int h, const ReqDesc& rq, unsigned char* smem) {
  constexpr int C = kAttnChunk;
  constexpr int RS = D + 1;                   // odd LDS row stride (floats)
  constexpr int V4 = C * D / 4 / 256;         // float4 loads per thread per matrix
  constexpr int QL = D / 64;                  // query elements per lane
  float* Ks = reinterpret_cast<float*>(smem);
  float* Vs = Ks + C * RS;
  float* qs = Vs + C * RS;
  float* ps = qs + 4 * D;

  const int nkeys = rq.L0 + rq.W;
  const int key0 = c * C;
  const int nk = min(C, nkeys - key0);
  const int g = h * p.n_kv / p.n_q;
  const int qcols = p.n_q * D;
  const float* kb = p.k_cache + (size_t)rq.slot * p.slot_stride + ((size_t)g * p.kv_cap + key0) * D;
  const float* vb = p.v_cache + (size_t)rq.slot * p.slot_stride + ((size_t)g * p.kv_cap + key0) * D;
  {
    float4 kv[V4], vv[V4];
#pragma unroll
    for (int t = 0; t < V4; ++t) {
      const int f = (t * 256 + threadIdx.x) * 4;   // element index in the chunk
      if (f < nk * D) {
        kv[t] = *reinterpret_cast<const float4*>(kb + f);
        vv[t] = *reinterpret_cast<const float4*>(vb + f);
      }
    }
#pragma unroll
    for (int t = 0; t < V4; ++t) {
      const int f = (t * 256 + threadIdx.x) * 4;
      if (f < nk * D) {
        const int j = f / D, dd = f - j * D;
        float* kd = Ks + j * RS + dd;
        float* vd = Vs + j * RS + dd;
        kd[0] = kv[t].x; kd[1] = kv[t].y; kd[2] = kv[t].z; kd[3] = kv[t].w;
        vd[0] = vv[t].x; vd[1] = vv[t].y; vd[2] = vv[t].z; vd[3] = vv[t].w;
      }
    }
  }

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = lane & (C - 1), half = lane >> 5;
  float* qw = qs + wave * D;
  float* pw = ps + wave * C;
  // first row of this wave at or after the chunk start
  int i = wave;
  while (i < rq.W && rq.L0 + i < key0) i += 4;
  float qn[QL];
  if (i < rq.W) {
#pragma unroll
    for (int t = 0; t < QL; ++t) qn[t] = p.q[(size_t)(rq.row_start + i) * qcols + h * D + t * 64 + lane];
  }
  __syncthreads();
  for (; i < rq.W; i += 4) {
    const int pos = rq.L0 + i;
    const int row = rq.row_start + i;
#pragma unroll
    for (int t = 0; t < QL; ++t) qw[t * 64 + lane] = qn[t];
    if (i + 4 < rq.W) {
#pragma unroll
      for (int t = 0; t < QL; ++t) qn[t] = p.q[(size_t)(row + 4) * qcols + h * D + t * 64 + lane];
    }
    __builtin_amdgcn_wave_barrier();
    const bool valid = j < nk && key0 + j <= pos;
    float a = 0.0f;
    if (j < nk) {
      const float* kr = Ks + j * RS + half * (D / 2);
      const float* qh = qw + half * (D / 2);
#pragma unroll 8
      for (int dd = 0; dd < D / 2; ++dd) a += qh[dd] * kr[dd];
    }
    a += __shfl_xor(a, 32);  // both halves: same sum (commutative)
    const float s = valid ? a * p.scale : -INFINITY;
    const float mx = wave_max(s);
    const float pj = valid ? expf(s - mx) : 0.0f;
    const float l = wave_sum(half == 0 ? pj : 0.0f);
    if (half == 0) pw[j] = pj;
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int t = 0; t < QL; ++t) {
      const int dd = t * 64 + lane;
      float o = 0.0f;
      for (int jj = 0; jj < nk; ++jj) o += pw[jj] * Vs[jj * RS + dd];
      st<COH>(p.pacc + (((size_t)c * kMaxRows + row) * p.n_q + h) * D + dd, o);
    }
    if (lane == 0) {
      st<COH>(p.pml + (((size_t)c * kMaxRows + row) * p.n_q + h) * 2, mx);
      st<COH>(p.pml + (((size_t)c * kMaxRows + row) * p.n_q + h) * 2 + 1, l);
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// Merge of row `row`'s chunks for head h by D threads starting at thread t0:
// chunk weights exp(m_c - max m) go through LDS (sm, sl: kMaxChunks floats
// each), then each thread sums its dimension over the chunks in ascending
// order with the loads issued in batches.  `sync` synchronises the threads
// that share it; with valid = false the threads only join those syncs.

template <bool BF, int D, bool COH, class Sync>
__device__ void attn_merge_row(const AttnArgs& p, int row, int h, int t0, float* sm, float* sl, Sync&& sync,
                               bool valid = true) {
  constexpr int kB = 8;
  const int dd = threadIdx.x - t0;
  const RowDesc rd = p.rows[row];
  const int nc = valid ? rd.pos / kAttnChunk + 1 : 0;
  auto ld = [](const float* q) { if constexpr (COH) return ld_coherent(q); else return *q; };
  for (int c = dd; c < nc; c += D) {
    const size_t o = ((size_t)c * kMaxRows + row) * p.n_q + h;
    sm[c] = ld(p.pml + o * 2);
    sl[c] = ld(p.pml + o * 2 + 1);
  }
  sync();
  float mx = -INFINITY;
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, sm[c]);
  sync();
  for (int c = dd; c < nc; c += D) sm[c] = expf(sm[c] - mx);
  sync();
  float L = 0.0f, a = 0.0f;
  for (int c0 = 0; c0 < nc; c0 += kB) {
    float v[kB];
#pragma unroll
    for (int b = 0; b < kB; ++b)
      if (c0 + b < nc) v[b] = ld(p.pacc + (((size_t)(c0 + b) * kMaxRows + row) * p.n_q + h) * D + dd);
#pragma unroll
    for (int b = 0; b < kB; ++b)
      if (c0 + b < nc) {
        L += sl[c0 + b] * sm[c0 + b];
        a += v[b] * sm[c0 + b];
      }
  }
  if (valid) store_act<BF, COH>(p.out, p.out_plane, (size_t)row * p.n_q * D + h * D + dd, a / L);
}

// ---------------------------------------------------------------------------
// Arg-max of row `row` over the LM head's per-group partials (256 threads):
// larger value wins, equal values keep the lower token id; *bad is set for a
// non-finite logit.  s4f / s4i: 4-entry LDS scratch.

template <bool COH>
__device__ void argmax_row(const float* amax_val, const int* amax_idx, int n_groups, int row, int* tok,
                           int* bad, float* s4f, int* s4i) {
  constexpr int kPer = 8;   // groups per thread, loads in flight together
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  bool b = false;
  for (int g0 = 0; g0 < n_groups; g0 += 256 * kPer) {
    float v[kPer];
    int id[kPer];
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int g = g0 + t * 256 + tid;
      if (g < n_groups) {
        if constexpr (COH) {
          v[t] = ld_coherent(amax_val + g * kMaxRows + row);
          id[t] = ld_coherent(amax_idx + g * kMaxRows + row);
        } else {
          v[t] = amax_val[g * kMaxRows + row];
          id[t] = amax_idx[g * kMaxRows + row];
        }
      }
    }
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int g = g0 + t * 256 + tid;
      if (g < n_groups) {
        if (!isfinite(v[t])) b = true;
        else if (v[t] > best || (v[t] == best && id[t] < bi)) { best = v[t]; bi = id[t]; }
      }
    }
  }
  wave_argmax(best, bi);
  const bool wb = __ballot(b) != 0;
  if (lane == 0) { s4f[wave] = best; s4i[wave] = bi | (wb ? 0x80000000 : 0); }
  __syncthreads();
  if (tid == 0) {
    float bv = s4f[0];
    int bx = s4i[0] & 0x7fffffff, bb = s4i[0] < 0;
    for (int w = 1; w < 4; ++w) {
      const int iw = s4i[w] & 0x7fffffff;
      if (s4f[w] > bv || (s4f[w] == bv && iw < bx)) { bv = s4f[w]; bx = iw; }
      bb |= s4i[w] < 0;
    }
    *tok = bx;
    *bad = bb | !isfinite(bv);
  }
  __syncthreads();
}

// Greedy verification of one request from its rows' greedy tokens
// (Section 4.2; Appendix C.2): accepted = first row i < W-1 whose greedy
// token differs from its candidate (W-1 if none); the correction is the
// greedy token of row `accepted`.
template <class TokAt>
__device__ StepOut verify_request(const RowDesc* rows, const ReqDesc& rq, TokAt&& tok_at, int bad) {
  int a = 0;
  while (a < rq.W - 1 && rows[rq.row_start + a].cmp == tok_at(rq.row_start + a)) ++a;
  return StepOut{a, tok_at(rq.row_start + a), bad, 0};
}

}  // namespace as2d
