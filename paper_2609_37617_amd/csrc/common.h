// Device helpers shared by the per-operation kernels (kernels.hip) and the
// persistent step kernel (step.hip): number formats, MFMA steps, memory
// access flavours and wave reductions.
#pragma once
#include <math.h>

#include "kernels.h"

namespace as2d {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// element formats

// bf16 nearest to f, ties to even (one v_cvt_pk_bf16_f32 on gfx950; NaN stays NaN).
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

template <bool BF> struct ET;
template <> struct ET<true> { typedef uint16_t T; static constexpr int PER16 = 8; };
template <> struct ET<false> { typedef float T; static constexpr int PER16 = 4; };

__device__ __forceinline__ float to_f(uint16_t v) { return bf2f(v); }
__device__ __forceinline__ float to_f(float v) { return v; }

// ---------------------------------------------------------------------------
// Global-memory views of device pointers.  A pointer the compiler cannot
// trace to a kernel argument (one read from a device-side argument array)
// is generic, and generic (flat) accesses are counted on both the vector
// memory and the LDS counters, so every LDS wait would also wait for the
// weight prefetch.  Accesses through these views are global instructions.
template <class T> using gmem_t = __attribute__((address_space(1))) T;
template <class T> __device__ __forceinline__ gmem_t<T>* gmem(T* p) { return (gmem_t<T>*)p; }
template <class T> __device__ __forceinline__ const gmem_t<T>* gmem(const T* p) { return (const gmem_t<T>*)p; }

// Plain 16-byte load (activation fragments).
__device__ __forceinline__ uint4 ldg(const uint4* p) {
  const u32x4 v = *gmem(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ldg(const float4* p) {
  const f4 v = *gmem(reinterpret_cast<const f4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float2 ldg(const float2* p) {
  const f2 v = *gmem(reinterpret_cast<const f2*>(p));
  return make_float2(v.x, v.y);
}
template <class V> __device__ __forceinline__ V ldg(const V* p) { return *gmem(p); }

// ---------------------------------------------------------------------------
// Stores of values other workgroups read.  COH = true: inside one kernel,
// possibly from another XCD (whose L2 is not coherent with the writer's):
// agent-scope stores that write through the L2.  COH = false: read only by
// later kernels (kernel boundaries make them visible).

template <bool COH, typename V> __device__ __forceinline__ void st(V* p, V v) {
  if constexpr (COH)
    __hip_atomic_store(gmem(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *gmem(p) = v;
}
template <typename V> __device__ __forceinline__ V ld_coherent(const V* p) {
  return __hip_atomic_load(gmem(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wider reads with the cache policy of ld_coherent (sc1: past this XCD's
// L2), through a raw buffer descriptor of the allocation's base: 8 or 16
// bytes at byte offset `off` (< 2^31, aligned to the access size).  For a
// lane that reads several consecutive floats another workgroup of the same
// launch stored with agent-scope stores.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}
constexpr int kCPolSC1 = 16;   // cache-policy bits of the buffer instructions: sc1
__device__ __forceinline__ float4 ld_coherent4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCPolSC1);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
}
__device__ __forceinline__ float2 ld_coherent2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCPolSC1);
  return make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
}

// Index of element (m, k) of an activation operand with K columns in MFMA
// fragment order: one block of 16 rows x KE elements (one k-step of one
// 16-row tile, 1 KiB) after another, tiles outer, k-steps inner; inside a
// block the 16 rows are row-major, so the rows a pass uses are a prefix of
// the block (rows past M need not be loaded).
template <bool BF> __host__ __device__ __forceinline__ size_t frag_index(int m, int k, int K) {
  constexpr int KE = 4 * ET<BF>::PER16;
  return (size_t)(m >> 4) * 16 * K + (size_t)(k / KE) * 16 * KE + (size_t)(m & 15) * KE + (k % KE);
}
// 16-byte unit of a block that lane l feeds to the MFMA (row l % 16, k-slice l / 16).
__device__ __forceinline__ int frag_lane_unit(int lane) { return (lane & 15) * 4 + (lane >> 4); }
// The same for a row tile with `rows` valid rows: lanes of the rows past
// them read row 0's unit (a line the wave loads anyway), so the load needs
// no branch and fetches no extra line; those lanes only feed output rows
// that are never stored.
__device__ __forceinline__ int frag_lane_unit_clamped(int lane, int rows) {
  return ((lane & 15) < rows ? (lane & 15) * 4 : 0) + (lane >> 4);
}

// Activation planes (kernels.h): store value v at element i.
template <bool BF, bool COH> __device__ __forceinline__ void store_act(void* base, long long plane, size_t i, float v) {
  if constexpr (BF) {
    uint16_t* b = static_cast<uint16_t*>(base);
    const uint16_t hi = f2bf(v);
    st<COH>(b + i, hi);
    st<COH>(b + i + plane, f2bf(v - bf2f(hi)));
  } else {
    st<COH>(static_cast<float*>(base) + i, v);
  }
}

// N consecutive elements v[0..N) at elements i .. i + N - 1 of the
// activation planes, which the caller guarantees lie in one k-step block
// (so they are contiguous in memory) with i a multiple of N (N = 4 or 8).
template <bool BF, bool COH, int N>
__device__ __forceinline__ void store_act_run(void* base, long long plane, size_t i, const float* v) {
  static_assert(N == 2 || N == 4 || N == 8, "run of 2, 4 or 8 elements");
  if constexpr (BF) {
    uint32_t hw[N / 2], lw[N / 2];
#pragma unroll
    for (int t = 0; t < N / 2; ++t) {
      const uint16_t h0 = f2bf(v[2 * t]), h1 = f2bf(v[2 * t + 1]);
      hw[t] = h0 | ((uint32_t)h1 << 16);
      lw[t] = f2bf(v[2 * t] - bf2f(h0)) | ((uint32_t)f2bf(v[2 * t + 1] - bf2f(h1)) << 16);
    }
    uint32_t* hp = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(base) + i);
    uint32_t* lp = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(base) + i + plane);
    if constexpr (COH) {
#pragma unroll
      for (int t = 0; t < N / 2; ++t) {
        st<true>(hp + t, hw[t]);
        st<true>(lp + t, lw[t]);
      }
    } else if constexpr (N == 8) {
      *gmem(reinterpret_cast<u32x4*>(hp)) = u32x4{hw[0], hw[1], hw[2], hw[3]};
      *gmem(reinterpret_cast<u32x4*>(lp)) = u32x4{lw[0], lw[1], lw[2], lw[3]};
    } else if constexpr (N == 2) {
      *gmem(hp) = hw[0];
      *gmem(lp) = lw[0];
    } else {
      *gmem(reinterpret_cast<u32x2*>(hp)) = u32x2{hw[0], hw[1]};
      *gmem(reinterpret_cast<u32x2*>(lp)) = u32x2{lw[0], lw[1]};
    }
  } else {
    float* fp = static_cast<float*>(base) + i;
    if constexpr (COH) {
#pragma unroll
      for (int t = 0; t < N; ++t) st<true>(fp + t, v[t]);
    } else if constexpr (N == 2) {
      *gmem(reinterpret_cast<f2*>(fp)) = f2{v[0], v[1]};
    } else {
#pragma unroll
      for (int t = 0; t < N; t += 4) *gmem(reinterpret_cast<f4*>(fp + t)) = f4{v[t], v[t + 1], v[t + 2], v[t + 3]};
    }
  }
}

// Wait until this wave's memory operations (its stores included) have been
// performed.
// Reads a struct that no thread writes while the kernel runs (per-layer
// arguments, request descriptors) through the constant address space: the
// fields arrive by scalar loads in scalar registers, so no later wait on
// the vector memory counter (which covers the weight prefetch) is needed
// for them.
template <class T> __device__ __forceinline__ T load_invariant(const T* p) {
  static_assert(sizeof(T) % 4 == 0 && alignof(T) >= 4, "copied as 32-bit words");
  T out;
  const __attribute__((address_space(4))) uint32_t* src = (const __attribute__((address_space(4))) uint32_t*)p;
  uint32_t* dst = reinterpret_cast<uint32_t*>(&out);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) dst[i] = src[i];
  return out;
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// The same wait through the compiler's own instruction (s_waitcnt vmcnt(0),
// expcnt and lgkmcnt left alone), so that its wait placement knows that every
// earlier vector memory operation has completed: a loop can then hold a
// second set of loads in flight without the counter's 63-entry limit making
// the compiler wait for everything.
__device__ __forceinline__ void wait_vmem_counted() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Agent-scope counter increment; returns the previous value.
__device__ __forceinline__ int counter_add(int* c, int v) {
  return __hip_atomic_fetch_add(gmem(c), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// MFMA steps.  16 bytes of A (row m = lane%16) times 16 bytes of B (column
// n = lane%16), accumulated into the 16x16 tile: lane holds rows
// 4*(lane/16)+i, column lane%16.  Lane group g = lane/16 carries the
// k-slice [g*PER16, (g+1)*PER16) of the step in both operands.

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

// Streaming (non-temporal) 16-byte load of weight tiles: read once per pass.
__device__ __forceinline__ uint4 ldw(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(gmem(reinterpret_cast<const u32x4*>(p)));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Split-K partials cross workgroups (and XCDs) inside one kernel: written
// and read with agent-scope accesses, so no fence has to write back or
// invalidate a whole L2.
__device__ __forceinline__ void store_partial(float* p, float v) { st<true>(p, v); }
__device__ __forceinline__ float load_partial(const float* p) { return ld_coherent(p); }

// Workgroup barrier ordering LDS only: outstanding global loads (the weight
// prefetch) stay in flight across it.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Fixed-pattern wave reductions on cross-lane data movement that does not
// go through LDS: DPP (pairs and quads, then mirrors of 8 and 16 lanes),
// a swizzle across the 16-lane rows of each half and, for the whole wave,
// the two halves read into scalar registers.  Each step adds the same two
// values on both partner lanes, so every lane (of the half, or of the
// wave) ends with the same bits.
template <int CTRL> __device__ __forceinline__ float dpp_get(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;         // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;         // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // lane i of 8 <- lane 7 - i
constexpr int kDppMirror = 0x140;      // lane i of 16 <- lane 15 - i
__device__ __forceinline__ float swizzle_xor16(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}
template <class Op> __device__ __forceinline__ float half_reduce(float v, Op op) {
  v = op(v, dpp_get<kDppXor1>(v));
  v = op(v, dpp_get<kDppXor2>(v));
  v = op(v, dpp_get<kDppHalfMirror>(v));
  v = op(v, dpp_get<kDppMirror>(v));
  return op(v, swizzle_xor16(v));
}
__device__ __forceinline__ float lane_value(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}
// Sum / max over each half-wave (lanes 0-31 and 32-63 separately).
__device__ __forceinline__ float half_sum(float v) {
  return half_reduce(v, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ float wave_sum(float v) {
  v = half_sum(v);
  return lane_value(v, 0) + lane_value(v, 32);
}
__device__ __forceinline__ float wave_max(float v) {
  v = half_reduce(v, [](float a, float b) { return fmaxf(a, b); });
  return fmaxf(lane_value(v, 0), lane_value(v, 32));
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
// The same over each half-wave (lanes 0-31 and 32-63 separately).
__device__ __forceinline__ void half_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 16; o > 0; o >>= 1) {
    float ov = __shfl_xor(v, o);
    int oi = __shfl_xor(i, o);
    if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
  }
}

// GEMM tile constants
constexpr int kPrefetchDirect = 4; // k-steps of weights and A in flight per wave (A direct)
constexpr int kFStride = 132;      // floats per row of the staged path's epilogue tile
constexpr int kFRows = 64;         // rows per epilogue pass of the staged path
constexpr int kStagedLds = 147456; // bytes of A staging (two buffers), staged path

}  // namespace as2d
