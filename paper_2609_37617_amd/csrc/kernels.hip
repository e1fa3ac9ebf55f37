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

// Activation planes (see kernels.h): store value v at element i.
template <bool BF> __device__ __forceinline__ void store_act(void* base, long long plane, size_t i, float v);
template <> __device__ __forceinline__ void store_act<true>(void* base, long long plane, size_t i, float v) {
  uint16_t* b = static_cast<uint16_t*>(base);
  const uint16_t hi = f2bf(v);
  b[i] = hi;
  b[i + plane] = f2bf(v - bf2f(hi));
}
template <> __device__ __forceinline__ void store_act<false>(void* base, long long, size_t i, float v) {
  static_cast<float*>(base)[i] = v;
}

// One k-step of one 16-row A tile: bf16 models carry (hi, lo), float32 one part.
struct AFrag {
  uint4 h, l;
};
template <bool BF> __device__ __forceinline__ f4 mma_a(const AFrag& a, uint4 b, f4 acc) {
  if constexpr (BF) {
    acc = mma_step<true>(a.h, b, acc);
    acc = mma_step<true>(a.l, b, acc);
  } else {
    acc = mma_step<false>(a.h, b, acc);
  }
  return acc;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// Streaming (non-temporal) 16-byte load of weight tiles: read once per pass.
__device__ __forceinline__ uint4 ldw(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Split-K partials cross workgroups (and XCDs, whose L2s are not coherent
// with each other) inside one kernel.  They are written and read with
// agent-scope atomic accesses, which bypass the non-coherent caching, so
// no fence has to write back or invalidate the whole L2.
__device__ __forceinline__ void store_partial(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_partial(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until this wave's memory operations, including the partial stores,
// have been performed.
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

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
// staging rows, the planes of x * g for the first RMSNorm (gain g), and
// per-row sum-of-squares partials over 128-column groups.  Each thread
// moves 8 consecutive elements per pass; every pass's loads are issued
// before any is used.

template <bool BF>
__global__ __launch_bounds__(256) void embed_kernel(const RowDesc* __restrict__ rows,
                                                    const typename ET<BF>::T* __restrict__ embed,
                                                    const typename ET<BF>::T* __restrict__ audio,
                                                    int H, const float* __restrict__ gain,
                                                    float* __restrict__ x, float* __restrict__ sumsq,
                                                    void* __restrict__ xg, long long xg_plane) {
  using T = typename ET<BF>::T;
  constexpr int kPer = 8, kPasses = 4;   // H <= 256 * 8 * 4
  extern __shared__ float srow[];
  const int m = blockIdx.x;
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
        x[(size_t)m * H + c0 + t] = v[ps][t];
        store_act<BF>(xg, xg_plane, (size_t)m * H + c0 + t, v[ps][t] * gain[c0 + t]);
        srow[c0 + t] = v[ps][t];
      }
    }
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
                        int H, const float* gain, float* x, float* sumsq, void* xg, long long xg_plane,
                        hipStream_t s) {
  if (H > 256 * 8 * 4 || H % 128) return hipErrorInvalidValue;
  const size_t lds = (size_t)H * sizeof(float);
  if (bf16)
    embed_kernel<true><<<M, 256, lds, s>>>(rows, (const uint16_t*)embed, (const uint16_t*)audio, H, gain,
                                           x, sumsq, xg, xg_plane);
  else
    embed_kernel<false><<<M, 256, lds, s>>>(rows, (const float*)embed, (const float*)audio, H, gain, x,
                                            sumsq, xg, xg_plane);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight-streaming GEMM  Y[M][N] = A[M][K] * W[N][K]^T  for small M.
//
// Workgroup = 4 waves over one 128-column group and one k-split; wave w
// owns the tile pair 4*group + w.  Each k-step a wave loads its two 1 KiB
// weight tiles (fully coalesced, non-temporal) and the A fragments of the
// same k-step, U steps ahead of their use.  Up to two 16-row tiles of A
// come straight from the L2-resident activation planes; larger M stages A
// through LDS in chunks.  Both paths issue the same MFMA sequence per row,
// so a row's result does not depend on M.  With KS > 1 each split writes a
// float32 partial and the last workgroup of a column group (device-scope
// counter) sums the partials in split order and runs the fused epilogue.

constexpr int kPrefetch = 4;
constexpr int kFStride = 132;      // floats per row of the epilogue tile
constexpr int kFRows = 64;         // rows per epilogue pass
constexpr int kDirectMT = 2;       // largest M-tile count loading A directly
constexpr int kLdsBudget = 61440;  // bytes of A staging
constexpr int kFixupBatch = 1;     // elements per thread with loads in flight in the split-K fixup

__host__ __device__ inline int lds_row_stride(int chunk_kt) {
  return ((chunk_kt * 64 + 127) / 128) * 128 + 16;
}

template <bool BF, int EPI>
__device__ void epilogue_rows(const GemmArgs& p, float* F, int group, int r0, int r1) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int N = p.N;
  if constexpr (EPI == EPI_RESID) {
    // x += Y; planes of x * g for the next RMSNorm; sum of squares of x
    for (int idx = tid; idx < (r1 - r0) * 128; idx += 256) {
      const int m = r0 + (idx >> 7), c = idx & 127;
      const int n = group * 128 + c;
      const size_t o = (size_t)m * N + n;
      const float v = p.x[o] + F[(m - r0) * kFStride + c];
      p.x[o] = v;
      store_act<BF>(p.out, p.out_plane, o, v * p.gain_next[n]);
      F[(m - r0) * kFStride + c] = v;
    }
    lds_sync();
    for (int m = r0 + wave; m < r1; m += 4) {
      const float v0 = F[(m - r0) * kFStride + lane], v1 = F[(m - r0) * kFStride + 64 + lane];
      const float s = wave_sum(v0 * v0 + v1 * v1);
      if (lane == 0) p.sumsq_out[group * kMaxRows + m] = s;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int F2 = N / 2;
    for (int idx = tid; idx < (r1 - r0) * 64; idx += 256) {
      const int m = r0 + (idx >> 6), c = idx & 63;
      const float g = F[(m - r0) * kFStride + c], u = F[(m - r0) * kFStride + 64 + c];
      store_act<BF>(p.out, p.out_plane, (size_t)m * F2 + group * 64 + c, g / (1.0f + expf(-g)) * u);
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
          p.k_cache[(size_t)rd.slot * p.slot_stride + ((size_t)kvh * p.kv_cap + rd.pos) * d + dd] = v;
        }
      } else {
        const int kvh = (n - qk_cols) / d;
        p.v_cache[(size_t)rd.slot * p.slot_stride + ((size_t)kvh * p.kv_cap + rd.pos) * d + dd] = v;
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
  constexpr int KE = 4 * PER16;           // elements per k-step
  constexpr bool kDirect = MT <= kDirectMT;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ float s_scale[kMaxRows];
  __shared__ int s_last;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int group = blockIdx.x / p.KS, split = blockIdx.x - group * p.KS;
  const int kt0 = split * p.ktps;
  const int kt1 = min(p.KT, kt0 + p.ktps);
  const int M = p.M, K = p.K;

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
    // stale data that only reaches output rows that are never stored)
    const T* abase = (const T*)p.A + (size_t)(lane & 15) * K + (lane >> 4) * PER16;
    auto load = [&](int kt, uint4(&bb)[2], AFrag(&af)[MT]) {
      bb[0] = ldw(wp + (size_t)kt * 128);
      bb[1] = ldw(wp + (size_t)kt * 128 + 64);
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
    for (int u = 0; u < kPrefetch; ++u) load(kt0 + min(u, n - 1), b[u], af[u]);
    int i = 0;
    for (; i + 2 * kPrefetch <= n; i += kPrefetch) {
#pragma unroll
      for (int u = 0; u < kPrefetch; ++u) {
        step(b[u], af[u]);
        load(kt0 + i + u + kPrefetch, b[u], af[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) {
      if (i + u < n) {
        step(b[u], af[u]);
        if (i + u + kPrefetch < n) load(kt0 + i + u + kPrefetch, b[u], af[u]);
      }
    }
    i += kPrefetch;
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u)
      if (i + u < n) step(b[u], af[u]);
  } else {
    // stage the A planes of `chunk_kt` k-steps in LDS (hi region, then lo)
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
    if (tid == 0)
      s_last = __hip_atomic_fetch_add(&p.counters[group], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
               p.KS - 1;
    __syncthreads();
    if (!s_last) return;
    if (tid == 0) p.counters[group] = 0;  // ready for the next launch
    for (int r0 = 0; r0 < M; r0 += kFRows) {
      const int r1 = min(M, r0 + kFRows);
      // every load of a batch of elements is issued before any is summed;
      // each element is still summed in split order
      const int nel = (r1 - r0) * 128;
      for (int e0 = 0; e0 < nel; e0 += 256 * kFixupBatch) {
        float v[kFixupBatch][kMaxSplits];
#pragma unroll
        for (int b = 0; b < kFixupBatch; ++b) {
          const int idx = e0 + b * 256 + tid;
          const int m = r0 + (idx >> 7), c = idx & 127;
#pragma unroll
          for (int sp = 0; sp < kMaxSplits; ++sp)
            if (idx < nel && sp < p.KS)
              v[b][sp] = load_partial(&p.part[((size_t)sp * M + m) * p.N + group * 128 + c]);
        }
#pragma unroll
        for (int b = 0; b < kFixupBatch; ++b) {
          const int idx = e0 + b * 256 + tid;
          if (idx < nel) {
            const int m = r0 + (idx >> 7), c = idx & 127;
            float sum = 0.0f;
#pragma unroll
            for (int sp = 0; sp < kMaxSplits; ++sp)
              if (sp < p.KS) sum += v[b][sp];
            F[(m - r0) * kFStride + c] = AM == A_NORM ? sum * s_scale[m] : sum;
          }
        }
      }
      lds_sync();
      epilogue_rows<BF, EPI>(p, F, group, r0, r1);
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
      epilogue_rows<BF, EPI>(p, F, group, r0, r1);
      lds_sync();
    }
  }
}

template <bool BF, int AM, int EPI>
static hipError_t gemm_dispatch(const GemmArgs& a, hipStream_t s) {
  const int regions = BF ? 2 : 1;
  int chunk = a.ktps;
  while (chunk > 1 && regions * a.MT * 16 * lds_row_stride(chunk) > kLdsBudget) --chunk;
  int lds = kFRows * kFStride * 4;
  if (a.MT > kDirectMT) lds = max(lds, regions * a.MT * 16 * lds_row_stride(chunk));
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
// Workgroup (chunk c, query head h, request r): keys [32c, 32c + 32) of the
// request's float32 cache slot are staged in LDS; each wave takes the
// request's rows in turn (the next row's query is prefetched into
// registers).  For a row at position pos >= 32c it computes the chunk's
// softmax statistics (max m, sum l of exp(s - m)) and the unnormalised
// output sum_j exp(s_j - m) v_j over keys j <= pos; lane pairs (j, j + 32)
// each take half of the dot product of key j.  The merge kernel combines a
// row's chunks in ascending order.

template <bool BF, int D>
__global__ __launch_bounds__(256) void attn_chunk_kernel(const AttnArgs p) {
  constexpr int C = kAttnChunk;
  constexpr int RS = D + 1;                   // odd LDS row stride (floats)
  constexpr int V4 = C * D / 4 / 256;         // float4 loads per thread per matrix
  constexpr int QL = D / 64;                  // query elements per lane
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  float* Ks = reinterpret_cast<float*>(smem);
  float* Vs = Ks + C * RS;
  float* qs = Vs + C * RS;
  float* ps = qs + 4 * D;

  const int c = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
  const ReqDesc rq = p.reqs[r];
  const int nkeys = rq.L0 + rq.W;
  const int key0 = c * C;
  if (key0 >= nkeys) return;
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
      p.pacc[(((size_t)c * kMaxRows + row) * p.n_q + h) * D + dd] = o;
    }
    if (lane == 0) {
      p.pml[(((size_t)c * kMaxRows + row) * p.n_q + h) * 2] = mx;
      p.pml[(((size_t)c * kMaxRows + row) * p.n_q + h) * 2 + 1] = l;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// Merge of a row's chunks (workgroup per (head, row), thread per output
// dimension): chunk weights exp(m_c - max m) go through LDS, then each
// thread sums its dimension over the chunks in ascending order with the
// loads issued in batches.
template <bool BF, int D>
__global__ __launch_bounds__(D) void attn_merge_kernel(const AttnArgs p) {
  constexpr int kB = 8;
  __shared__ float sm[kMaxChunks], sl[kMaxChunks];
  const int h = blockIdx.x, row = blockIdx.y, dd = threadIdx.x;
  const RowDesc rd = p.rows[row];
  const int nc = rd.pos / kAttnChunk + 1;
  for (int c = dd; c < nc; c += D) {
    const size_t o = ((size_t)c * kMaxRows + row) * p.n_q + h;
    sm[c] = p.pml[o * 2];
    sl[c] = p.pml[o * 2 + 1];
  }
  __syncthreads();
  float mx = -INFINITY;
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, sm[c]);
  __syncthreads();
  for (int c = dd; c < nc; c += D) sm[c] = expf(sm[c] - mx);
  __syncthreads();
  float L = 0.0f, a = 0.0f;
  for (int c0 = 0; c0 < nc; c0 += kB) {
    float v[kB];
#pragma unroll
    for (int b = 0; b < kB; ++b)
      if (c0 + b < nc) v[b] = p.pacc[(((size_t)(c0 + b) * kMaxRows + row) * p.n_q + h) * D + dd];
#pragma unroll
    for (int b = 0; b < kB; ++b)
      if (c0 + b < nc) {
        L += sl[c0 + b] * sm[c0 + b];
        a += v[b] * sm[c0 + b];
      }
  }
  store_act<BF>(p.out, p.out_plane, (size_t)row * p.n_q * D + h * D + dd, a / L);
}

template <bool BF, int D>
static hipError_t attn_dispatch(const AttnArgs& a, int n_reqs, int max_chunks, hipStream_t s) {
  if (max_chunks > kMaxChunks) return hipErrorInvalidValue;
  const size_t lds = (2 * kAttnChunk * (D + 1) + 4 * D + 4 * kAttnChunk) * sizeof(float);
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
// Final arg-max over the LM head's per-group partials, one workgroup per
// verified row, then greedy verification (Section 4.2; Appendix C.2) by the
// last row of each request to finish: accepted = first row i < W-1 whose
// greedy token differs from its candidate (W-1 if none), correction =
// greedy token of row `accepted`.

__global__ __launch_bounds__(256) void finish_kernel(const RowDesc* __restrict__ rows,
                                                     const ReqDesc* __restrict__ reqs, int n_reqs,
                                                     const float* __restrict__ amax_val,
                                                     const int* __restrict__ amax_idx, int n_groups,
                                                     int* __restrict__ row_tok, int* __restrict__ row_bad,
                                                     int* __restrict__ counters, StepOut* __restrict__ out) {
  constexpr int kPer = 8;   // groups per thread, loads in flight together
  __shared__ float s_v[4];
  __shared__ int s_i[4], s_b[4], s_last;
  // which request / row this workgroup verifies
  int r = 0, i = blockIdx.x;
  while (r < n_reqs - 1 && i >= reqs[r].W) i -= reqs[r++].W;
  const ReqDesc rq = reqs[r];
  const int row = rq.row_start + i;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  bool bad = false;
  for (int g0 = 0; g0 < n_groups; g0 += 256 * kPer) {
    float v[kPer];
    int id[kPer];
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int g = g0 + t * 256 + tid;
      if (g < n_groups) {
        v[t] = amax_val[g * kMaxRows + row];
        id[t] = amax_idx[g * kMaxRows + row];
      }
    }
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int g = g0 + t * 256 + tid;
      if (g < n_groups) {
        if (!isfinite(v[t])) bad = true;
        else if (v[t] > best || (v[t] == best && id[t] < bi)) { best = v[t]; bi = id[t]; }
      }
    }
  }
  wave_argmax(best, bi);
  const bool wbad = __ballot(bad) != 0;
  if (lane == 0) { s_v[wave] = best; s_i[wave] = bi; s_b[wave] = wbad; }
  __syncthreads();
  if (tid == 0) {
    float bv = s_v[0];
    int bx = s_i[0], bb = s_b[0];
    for (int w = 1; w < 4; ++w) {
      if (s_v[w] > bv || (s_v[w] == bv && s_i[w] < bx)) { bv = s_v[w]; bx = s_i[w]; }
      bb |= s_b[w];
    }
    bb |= !isfinite(bv);
    __hip_atomic_store(&row_tok[row], bx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&row_bad[row], bb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    wait_vmem();
    s_last = __hip_atomic_fetch_add(&counters[r], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == rq.W - 1;
    if (s_last) {
      counters[r] = 0;  // ready for the next launch
      int a = 0, nan = 0;
      for (int q = 0; q < rq.W; ++q)
        nan |= __hip_atomic_load(&row_bad[rq.row_start + q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      while (a < rq.W - 1 && rows[rq.row_start + a].cmp ==
                                 __hip_atomic_load(&row_tok[rq.row_start + a], __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT))
        ++a;
      const int corr = __hip_atomic_load(&row_tok[rq.row_start + a], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      out[r] = StepOut{a, corr, nan, 0};
    }
  }
}

hipError_t launch_finish(const RowDesc* rows, const ReqDesc* reqs, int n_reqs, int n_rows,
                         const float* amax_val, const int* amax_idx, int n_groups, int* row_tok,
                         int* row_bad, int* counters, StepOut* out, hipStream_t s) {
  finish_kernel<<<n_rows, 256, 0, s>>>(rows, reqs, n_reqs, amax_val, amax_idx, n_groups, row_tok, row_bad,
                                       counters, out);
  return hipGetLastError();
}

}  // namespace as2d
