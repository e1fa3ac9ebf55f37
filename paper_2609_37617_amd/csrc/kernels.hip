// gfx950 kernels of the target verification step.
//
// Every row's arithmetic is independent of how many rows share the pass:
// GEMM k-splits depend only on the matrix shape, attention splits the key
// axis at fixed 64-key boundaries and merges them in order, and arg-max is
// exact.  A verification call over root + k candidates therefore computes,
// bit for bit, the logits and cache rows of k + 1 sequential target-only
// steps (the pathwise-equivalence requirement of Appendix C.4, met here
// numerically and not only up to masks).
#include "kernels.h"

#include <math.h>

namespace as2d {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------------------
// element helpers

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);                      // round to nearest even
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

template <bool BF> struct ET;
template <> struct ET<true> { typedef uint16_t T; static constexpr int PER16 = 8; };
template <> struct ET<false> { typedef float T; static constexpr int PER16 = 4; };

__device__ __forceinline__ float to_f(uint16_t v) { return bf2f(v); }
__device__ __forceinline__ float to_f(float v) { return v; }
template <bool BF> __device__ __forceinline__ typename ET<BF>::T from_f(float v);
template <> __device__ __forceinline__ uint16_t from_f<true>(float v) { return f2bf(v); }
template <> __device__ __forceinline__ float from_f<false>(float v) { return v; }

// 16 bytes of A (row m = lane%16) times 16 bytes of B (column n = lane%16),
// accumulated into the 16x16 tile: lane holds rows 4*(lane/16)+i, column
// lane%16.  Lane group g = lane/16 carries the k-slice [g*PER16, (g+1)*PER16)
// of the step in both operands.
template <bool BF> __device__ __forceinline__ f4 mma_step(uint4 a, uint4 b, f4 acc);
template <> __device__ __forceinline__ f4 mma_step<true>(uint4 a, uint4 b, f4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}
template <> __device__ __forceinline__ f4 mma_step<false>(uint4 a, uint4 b, f4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  return acc;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// Streaming (non-temporal) 16-byte load of weight tiles: read once per pass.
__device__ __forceinline__ uint4 ldw(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Workgroup barrier ordering LDS only: outstanding global loads (the weight
// prefetch) stay in flight across it.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Fixed-pattern wave reductions; callers use lane 0's result.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
// (value, index) arg-max: larger value wins, equal values keep the lower index.
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float ov = __shfl_xor(v, o);
    int oi = __shfl_xor(i, o);
    if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
  }
}

// ---------------------------------------------------------------------------
// Weight packing: row-major [N][K] -> 1 KiB tiles in the order one wave
// streams them.  Tile (nt, kt) covers rows [16 nt, 16 nt + 16) and k-step kt;
// lane l holds row 16 nt + l%16, elements [kt*KE + (l/16)*PER16, +PER16).
// Tiles of a wave's pair (nt = 2 tp + j) are adjacent per k-step:
//   index ((tp * KT + kt) * 2 + j) * 64 + lane.
// remap_gate_up: virtual row v of the fused gate/up matrix ([gate; up] in
// src, 2F rows) takes gate row 64 g + c for c < 64 and up row 64 g + c - 64
// otherwise (g = v / 128, c = v % 128), so each 128-column group holds the
// gate and up columns of the same 64 FFN units.

template <bool BF>
__global__ void pack_kernel(const typename ET<BF>::T* __restrict__ src, uint4* __restrict__ dst,
                            int N, int K, int remap, int F) {
  constexpr int PER16 = ET<BF>::PER16;
  constexpr int KE = 4 * PER16;
  const int KT = K / KE;
  const long long total = (long long)(N / 16) * KT * 64;  // 64 lanes x 16 B per 16-row tile
  for (long long idx = blockIdx.x * (long long)blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int lane = (int)(idx & 63);
    const long long t = idx >> 6;
    const int j = (int)(t & 1);
    const long long u = t >> 1;
    const int kt = (int)(u % KT);
    const int tp = (int)(u / KT);
    const int nt = tp * 2 + j;
    int row = nt * 16 + (lane & 15);
    if (remap) {
      const int g = row / 128, c = row % 128;
      row = c < 64 ? 64 * g + c : F + 64 * g + (c - 64);
    }
    const int k0 = kt * KE + (lane >> 4) * PER16;
    dst[idx] = *reinterpret_cast<const uint4*>(src + (size_t)row * K + k0);
  }
}

hipError_t launch_pack(bool bf16, const void* src, uint4* dst, int N, int K, int remap, int F,
                       hipStream_t s) {
  const int threads = 256, blocks = 4096;
  if (bf16)
    pack_kernel<true><<<blocks, threads, 0, s>>>((const uint16_t*)src, dst, N, K, remap, F);
  else
    pack_kernel<false><<<blocks, threads, 0, s>>>((const float*)src, dst, N, K, remap, F);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Embedding gather: residual rows x (float32) from token embeddings or audio
// staging rows, plus per-row sum-of-squares partials over 128-column groups
// for the first RMSNorm.

template <bool BF>
__global__ __launch_bounds__(256) void embed_kernel(const RowDesc* __restrict__ rows,
                                                    const typename ET<BF>::T* __restrict__ embed,
                                                    const typename ET<BF>::T* __restrict__ audio,
                                                    int H, float* __restrict__ x,
                                                    float* __restrict__ sumsq) {
  extern __shared__ float srow[];
  const int m = blockIdx.x;
  const RowDesc rd = rows[m];
  const typename ET<BF>::T* src =
      rd.token >= 0 ? embed + (size_t)rd.token * H : audio + (size_t)rd.src * H;
  for (int c = threadIdx.x; c < H; c += 256) {
    const float v = to_f(src[c]);
    x[(size_t)m * H + c] = v;
    srow[c] = v;
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int g = wave; g < H / 128; g += 4) {
    const float v0 = srow[g * 128 + lane], v1 = srow[g * 128 + 64 + lane];
    const float s = wave_sum(v0 * v0 + v1 * v1);
    if (lane == 0) sumsq[g * kMaxRows + m] = s;
  }
}

hipError_t launch_embed(bool bf16, const RowDesc* rows, int M, const void* embed, const void* audio,
                        int H, float* x, float* sumsq, hipStream_t s) {
  const size_t lds = (size_t)H * sizeof(float);
  if (bf16)
    embed_kernel<true><<<M, 256, lds, s>>>(rows, (const uint16_t*)embed, (const uint16_t*)audio, H,
                                           x, sumsq);
  else
    embed_kernel<false><<<M, 256, lds, s>>>(rows, (const float*)embed, (const float*)audio, H, x,
                                            sumsq);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight-streaming GEMM  Y[M][N] = A[M][K] * W[N][K]^T  for small M.
//
// Workgroup = 4 waves over one 128-column group and one k-split; wave w
// owns the tile pair 4*group + w.  A (all M rows of the split's K range,
// converted to the element type, RMSNorm applied when AM == A_NORM) is
// staged in LDS; the weight tiles stream from HBM with a U-deep register
// prefetch, one 1 KiB fully coalesced load per tile and k-step.  With
// KS > 1 each split writes a float32 partial and the last workgroup to
// finish a column group (device-scope counter) sums the partials in split
// order and runs the fused epilogue.

constexpr int kPrefetch = 4;
constexpr int kFStride = 132;      // floats per row of the epilogue tile
constexpr int kFRows = 64;         // rows per epilogue pass

__host__ __device__ inline int lds_row_stride(int chunk_kt) {
  return ((chunk_kt * 64 + 127) / 128) * 128 + 16;
}

int gemm_lds_bytes(bool, int MT, int chunk_kt) {
  const int a = MT * 16 * lds_row_stride(chunk_kt);
  const int f = kFRows * kFStride * 4;
  return a > f ? a : f;
}

template <bool BF, int EPI>
__device__ void epilogue_rows(const GemmArgs& p, const float* F, int group, int r0, int r1) {
  using T = typename ET<BF>::T;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int N = p.N;
  if constexpr (EPI == EPI_RESID) {
    // x += Y; then the sum of squares of the new x over this group's columns
    float* Fw = const_cast<float*>(F);
    for (int idx = tid; idx < (r1 - r0) * 128; idx += 256) {
      const int m = r0 + (idx >> 7), c = idx & 127;
      const size_t o = (size_t)m * N + group * 128 + c;
      const float v = p.x[o] + Fw[(m - r0) * kFStride + c];
      p.x[o] = v;
      Fw[(m - r0) * kFStride + c] = v;
    }
    lds_sync();
    for (int m = r0 + wave; m < r1; m += 4) {
      const float v0 = F[(m - r0) * kFStride + lane], v1 = F[(m - r0) * kFStride + 64 + lane];
      const float s = wave_sum(v0 * v0 + v1 * v1);
      if (lane == 0) p.sumsq_out[group * kMaxRows + m] = s;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    T* h = (T*)p.h_out;
    const int F2 = N / 2;
    for (int idx = tid; idx < (r1 - r0) * 64; idx += 256) {
      const int m = r0 + (idx >> 6), c = idx & 63;
      const float g = F[(m - r0) * kFStride + c], u = F[(m - r0) * kFStride + 64 + c];
      h[(size_t)m * F2 + group * 64 + c] = from_f<BF>(g / (1.0f + expf(-g)) * u);
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
          p.q_out[(size_t)m * q_cols + n] = v;
        } else {
          const int kvh = (n - q_cols) / d;
          T* kc = (T*)p.k_cache + (size_t)rd.slot * p.slot_stride +
                  ((size_t)kvh * p.kv_cap + rd.pos) * d + dd;
          *kc = from_f<BF>(v);
        }
      } else {
        const int kvh = (n - qk_cols) / d;
        T* vc = (T*)p.v_cache + (size_t)rd.slot * p.slot_stride +
                ((size_t)kvh * p.kv_cap + rd.pos) * d + dd;
        *vc = from_f<BF>(v);
      }
    }
  } else {  // EPI_ARGMAX
    for (int m = r0 + wave; m < r1; m += 4) {
      const float v0 = F[(m - r0) * kFStride + lane], v1 = F[(m - r0) * kFStride + 64 + lane];
      const int n0 = group * 128 + lane;
      if (p.logits) {
        p.logits[(size_t)m * N + n0] = v0;
        p.logits[(size_t)m * N + n0 + 64] = v1;
      }
      const bool bad = !(isfinite(v0) && isfinite(v1));
      float best = v0;
      int bi = n0;
      if (v1 > best) { best = v1; bi = n0 + 64; }
      wave_argmax(best, bi);
      const bool any_bad = __ballot(bad) != 0;
      if (lane == 0) {
        p.amax_val[group * kMaxRows + m] = any_bad ? __builtin_nanf("") : best;
        p.amax_idx[group * kMaxRows + m] = bi;
      }
    }
  }
}

template <bool BF, int MT, int AM, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmArgs p, const int chunk_kt) {
  using T = typename ET<BF>::T;
  constexpr int PER16 = ET<BF>::PER16;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ float s_scale[kMaxRows];
  __shared__ int s_last;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int group = blockIdx.x / p.KS, split = blockIdx.x - group * p.KS;
  const int kt0 = split * p.ktps;
  const int kt1 = min(p.KT, kt0 + p.ktps);
  const int M = p.M;
  const int stride = lds_row_stride(chunk_kt);

  if constexpr (AM == A_NORM) {
    for (int m = tid; m < M; m += 256) {
      float ss = 0.0f;
      for (int g = 0; g < p.n_norm_groups; ++g) ss += p.sumsq[g * kMaxRows + m];
      s_scale[m] = 1.0f / sqrtf(ss / (float)p.K + p.eps);
    }
    __syncthreads();
  }

  f4 acc[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt][0] = f4{0.f, 0.f, 0.f, 0.f};
    acc[mt][1] = f4{0.f, 0.f, 0.f, 0.f};
  }
  const uint4* wp = p.W + (size_t)(group * kWaves + wave) * p.KT * 128 + lane;
  const unsigned char* abase = smem + (lane & 15) * stride + (lane >> 4) * 16;

  for (int c0 = kt0; c0 < kt1; c0 += chunk_kt) {
    const int c1 = min(kt1, c0 + chunk_kt);
    const int n = c1 - c0;
    if (c0 != kt0) lds_sync();
    // stage A rows [0, 16 MT) x k-steps [c0, c1) as 16-byte units
    const int units = MT * 16 * n * 4;
    for (int u = tid; u < units; u += 256) {
      const int m = u / (n * 4), r = u - m * (n * 4);
      const int k = (c0 + (r >> 2)) * (4 * PER16) + (r & 3) * PER16;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (m < M) {
        if constexpr (AM == A_PLAIN) {
          val = *reinterpret_cast<const uint4*>((const T*)p.A + (size_t)m * p.K + k);
        } else {
          const float* xr = (const float*)p.A + (size_t)m * p.K + k;
          const float sc = s_scale[m];
          T e[PER16];
#pragma unroll
          for (int t = 0; t < PER16; ++t) e[t] = from_f<BF>(xr[t] * sc * p.gain[k + t]);
          val = *reinterpret_cast<const uint4*>(e);
        }
      }
      *reinterpret_cast<uint4*>(smem + m * stride + (r >> 2) * 64 + (r & 3) * 16) = val;
    }
    // weight prefetch for the first k-steps of this chunk (unconditional, so
    // the load order is the same on every path into the loop below)
    uint4 b[kPrefetch][2];
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      const size_t kp = (size_t)(c0 + min(u, n - 1)) * 128;
      b[u][0] = ldw(wp + kp);
      b[u][1] = ldw(wp + kp + 64);
    }
    lds_sync();
    auto step = [&](const uint4(&bb)[2], int ks) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const uint4 a = *reinterpret_cast<const uint4*>(abase + mt * 16 * stride + ks * 64);
        acc[mt][0] = mma_step<BF>(a, bb[0], acc[mt][0]);
        acc[mt][1] = mma_step<BF>(a, bb[1], acc[mt][1]);
      }
    };
    // steady state: every refill is in range, so the loop body has no
    // branches and the prefetch depth holds across iterations
    int i = 0;
    for (; i + 2 * kPrefetch <= n; i += kPrefetch) {
#pragma unroll
      for (int u = 0; u < kPrefetch; ++u) {
        step(b[u], i + u);
        const size_t kn = (size_t)(c0 + i + u + kPrefetch) * 128;
        b[u][0] = ldw(wp + kn);
        b[u][1] = ldw(wp + kn + 64);
      }
    }
    // tail: at most 2 * kPrefetch - 1 steps left
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      if (i + u < n) {
        step(b[u], i + u);
        if (i + u + kPrefetch < n) {
          const size_t kn = (size_t)(c0 + i + u + kPrefetch) * 128;
          b[u][0] = ldw(wp + kn);
          b[u][1] = ldw(wp + kn + 64);
        }
      }
    }
    i += kPrefetch;
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u)
      if (i + u < n) step(b[u], i + u);
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
          if (row < M) p.part[((size_t)split * M + row) * p.N + col] = acc[mt][j][i];
        }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = atomicAdd(&p.counters[group], 1) == p.KS - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (tid == 0) p.counters[group] = 0;
    for (int r0 = 0; r0 < M; r0 += kFRows) {
      const int r1 = min(M, r0 + kFRows);
      for (int idx = tid; idx < (r1 - r0) * 128; idx += 256) {
        const int m = r0 + (idx >> 7), c = idx & 127;
        float s = 0.0f;
        for (int sp = 0; sp < p.KS; ++sp) s += p.part[((size_t)sp * M + m) * p.N + group * 128 + c];
        F[(m - r0) * kFStride + c] = s;
      }
      lds_sync();
      epilogue_rows<BF, EPI>(p, F, group, r0, r1);
      lds_sync();
    }
  } else {
    lds_sync();  // A tiles no longer read
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
            if (row >= r0 && row < r1) F[(row - r0) * kFStride + col] = acc[mt][j][i];
          }
      lds_sync();
      epilogue_rows<BF, EPI>(p, F, group, r0, r1);
      lds_sync();
    }
  }
}

template <bool BF, int AM, int EPI>
static hipError_t gemm_dispatch(const GemmArgs& a, hipStream_t s) {
  int chunk = a.ktps;
  while (chunk > 1 && a.MT * 16 * lds_row_stride(chunk) > 61440) --chunk;
  const int lds = gemm_lds_bytes(BF, a.MT, chunk);
  const dim3 grid((a.N / kGroupCols) * a.KS), block(256);
  switch (a.MT) {
#define AS2D_MT(mt) \
  case mt: gemm_kernel<BF, mt, AM, EPI><<<grid, block, lds, s>>>(a, chunk); break;
    AS2D_MT(1) AS2D_MT(2) AS2D_MT(3) AS2D_MT(4) AS2D_MT(5) AS2D_MT(6) AS2D_MT(7) AS2D_MT(8) AS2D_MT(9)
#undef AS2D_MT
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(bool bf16, int amode, int epi, const GemmArgs& a, hipStream_t s) {
#define AS2D_G(bf, am, ep) \
  if (bf16 == bf && amode == am && epi == ep) return gemm_dispatch<bf, am, ep>(a, s);
  AS2D_G(true, A_NORM, EPI_QKV) AS2D_G(true, A_PLAIN, EPI_RESID) AS2D_G(true, A_NORM, EPI_SWIGLU)
  AS2D_G(true, A_NORM, EPI_ARGMAX)
  AS2D_G(false, A_NORM, EPI_QKV) AS2D_G(false, A_PLAIN, EPI_RESID) AS2D_G(false, A_NORM, EPI_SWIGLU)
  AS2D_G(false, A_NORM, EPI_ARGMAX)
#undef AS2D_G
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Block-causal grouped-query attention, split over the key axis.
//
// Workgroup (chunk c, query head h, request r): keys [64c, 64c + 64) of the
// request's cache slot are staged in LDS; each wave takes the request's rows
// in turn and computes, for a row at position pos >= 64c, the chunk's
// softmax statistics (max m, sum l of exp(s - m)) and the unnormalised
// output sum_j exp(s_j - m) v_j over keys j <= pos.  The merge kernel
// combines the chunks of a row in ascending order.

template <bool BF, int D>
__global__ __launch_bounds__(256) void attn_chunk_kernel(const AttnArgs p) {
  using T = typename ET<BF>::T;
  constexpr int RS = BF ? D + 2 : D + 1;  // LDS row stride (elements): odd dword stride
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* Ks = reinterpret_cast<T*>(smem);
  T* Vs = Ks + 64 * RS;
  float* qs = reinterpret_cast<float*>(smem + ((2 * 64 * RS * sizeof(T) + 15) / 16) * 16);
  float* ps = qs + 4 * D;

  const int c = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
  const ReqDesc rq = p.reqs[r];
  const int nkeys = rq.L0 + rq.W;
  const int key0 = c * kAttnChunk;
  if (key0 >= nkeys) return;
  const int nk = min(kAttnChunk, nkeys - key0);
  const int g = h * p.n_kv / p.n_q;
  const int qcols = p.n_q * D;
  const T* kb = (const T*)p.k_cache + (size_t)rq.slot * p.slot_stride + ((size_t)g * p.kv_cap + key0) * D;
  const T* vb = (const T*)p.v_cache + (size_t)rq.slot * p.slot_stride + ((size_t)g * p.kv_cap + key0) * D;
  for (int idx = threadIdx.x; idx < nk * D; idx += 256) {
    const int j = idx / D, dd = idx - j * D;
    Ks[j * RS + dd] = kb[idx];
    Vs[j * RS + dd] = vb[idx];
  }
  __syncthreads();

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float* qw = qs + wave * D;
  float* pw = ps + wave * 64;
  for (int i = wave; i < rq.W; i += 4) {
    const int pos = rq.L0 + i;
    if (pos < key0) continue;
    const int row = rq.row_start + i;
    for (int dd = lane; dd < D; dd += 64) qw[dd] = p.q[(size_t)row * qcols + h * D + dd];
    __builtin_amdgcn_wave_barrier();
    const bool valid = lane < nk && key0 + lane <= pos;
    float s = -INFINITY;
    if (valid) {
      float a = 0.0f;
      const T* kr = Ks + lane * RS;
#pragma unroll 8
      for (int dd = 0; dd < D; ++dd) a += qw[dd] * to_f(kr[dd]);
      s = a * p.scale;
    }
    const float mx = wave_max(s);
    const float pj = valid ? expf(s - mx) : 0.0f;
    const float l = wave_sum(pj);
    pw[lane] = pj;
    __builtin_amdgcn_wave_barrier();
    for (int dd = lane; dd < D; dd += 64) {
      float a = 0.0f;
      for (int j = 0; j < nk; ++j) a += pw[j] * to_f(Vs[j * RS + dd]);
      p.pacc[(((size_t)c * kMaxRows + row) * p.n_q + h) * D + dd] = a;
    }
    if (lane == 0) {
      p.pml[(((size_t)c * kMaxRows + row) * p.n_q + h) * 2] = mx;
      p.pml[(((size_t)c * kMaxRows + row) * p.n_q + h) * 2 + 1] = l;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <bool BF, int D>
__global__ void attn_merge_kernel(const AttnArgs p) {
  using T = typename ET<BF>::T;
  const int h = blockIdx.x, row = blockIdx.y, dd = threadIdx.x;
  const RowDesc rd = p.rows[row];
  const int nc = rd.pos / kAttnChunk + 1;
  float mx = -INFINITY;
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, p.pml[(((size_t)c * kMaxRows + row) * p.n_q + h) * 2]);
  float L = 0.0f, a = 0.0f;
  for (int c = 0; c < nc; ++c) {
    const size_t o = ((size_t)c * kMaxRows + row) * p.n_q + h;
    const float w = expf(p.pml[o * 2] - mx);
    L += p.pml[o * 2 + 1] * w;
    a += p.pacc[o * D + dd] * w;
  }
  ((T*)p.out)[(size_t)row * p.n_q * D + h * D + dd] = from_f<BF>(a / L);
}

template <bool BF, int D>
static hipError_t attn_dispatch(const AttnArgs& a, int n_reqs, int max_chunks, hipStream_t s) {
  using T = typename ET<BF>::T;
  constexpr int RS = BF ? D + 2 : D + 1;
  const size_t lds = ((2 * 64 * RS * sizeof(T) + 15) / 16) * 16 + (4 * D + 4 * 64) * sizeof(float);
  attn_chunk_kernel<BF, D><<<dim3(max_chunks, a.n_q, n_reqs), 256, lds, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_merge_kernel<BF, D><<<dim3(a.n_q, a.M), D, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_attention(bool bf16, const AttnArgs& a, int n_reqs, int max_chunks, hipStream_t s) {
  if (a.head_dim == 128) return bf16 ? attn_dispatch<true, 128>(a, n_reqs, max_chunks, s)
                                     : attn_dispatch<false, 128>(a, n_reqs, max_chunks, s);
  if (a.head_dim == 64) return bf16 ? attn_dispatch<true, 64>(a, n_reqs, max_chunks, s)
                                    : attn_dispatch<false, 64>(a, n_reqs, max_chunks, s);
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Final arg-max over the LM head's per-group partials and greedy
// verification (Section 4.2; Appendix C.2): accepted = first row i < W-1
// whose greedy token differs from its candidate (W-1 if none), correction =
// greedy token of row `accepted`.

__global__ __launch_bounds__(256) void finish_kernel(const RowDesc* __restrict__ rows,
                                                     const ReqDesc* __restrict__ reqs,
                                                     const float* __restrict__ amax_val,
                                                     const int* __restrict__ amax_idx, int n_groups,
                                                     int* __restrict__ row_tok, StepOut* __restrict__ out) {
  __shared__ int s_tok[32];
  __shared__ int s_bad[32];
  const ReqDesc rq = reqs[blockIdx.x];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int i = wave; i < rq.W; i += 4) {
    const int row = rq.row_start + i;
    float best = -INFINITY;
    int bi = 0x7fffffff;
    bool bad = false;
    for (int g = lane; g < n_groups; g += 64) {
      const float v = amax_val[g * kMaxRows + row];
      const int id = amax_idx[g * kMaxRows + row];
      if (!isfinite(v)) bad = true;
      else if (v > best || (v == best && id < bi)) { best = v; bi = id; }
    }
    wave_argmax(best, bi);
    const bool any_bad = (__ballot(bad) != 0) || !isfinite(best);
    if (lane == 0) {
      s_tok[i] = bi;
      s_bad[i] = any_bad;
      row_tok[row] = bi;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int bad = 0;
    for (int i = 0; i < rq.W; ++i) bad |= s_bad[i];
    int a = 0;
    while (a < rq.W - 1 && rows[rq.row_start + a].cmp == s_tok[a]) ++a;
    out[blockIdx.x] = StepOut{a, s_tok[a], bad, 0};
  }
}

hipError_t launch_finish(const RowDesc* rows, const ReqDesc* reqs, int n_reqs, const float* amax_val,
                         const int* amax_idx, int n_groups, int* row_tok, StepOut* out, hipStream_t s) {
  finish_kernel<<<n_reqs, 256, 0, s>>>(rows, reqs, amax_val, amax_idx, n_groups, row_tok, out);
  return hipGetLastError();
}

}  // namespace as2d
