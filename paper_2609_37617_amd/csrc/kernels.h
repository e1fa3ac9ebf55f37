// Internal interface between the C ABI (as2d.cpp) and the gfx950 kernels
// (kernels.hip).  Not installed; the public interface is include/as2d.h.
//
// Number formats.  Weights and the embedding table are stored in the model
// dtype (bf16 or float32).  Everything else is float32 in value: the
// residual stream, the KV cache, softmax and all accumulators.  A GEMM
// operand that is an activation is handed over as "planes": for bf16
// models two bf16 planes hi = bf16(a), lo = bf16(a - hi) (a = hi + lo to
// about 2^-17 relative), multiplied into the bf16 weights by two MFMAs;
// for float32 models a single float32 plane.  A plane holds [kMaxRows][K]
// elements in MFMA fragment order (frag_index in common.h): every 16-row
// tile and k-step is one contiguous 1 KiB block, read by one wave with one
// load.  The lo plane starts `plane` elements after the hi plane.
//
// Per-pair partials (sum of squares for RMSNorm, arg-max of the LM head)
// are row-major [row][N / 32], so the partials of one row are contiguous.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace as2d {

// GEMM tiling shared by the packer and the GEMM kernels.  The unit of
// output columns is a tile pair: 32 columns, two 16-column MFMA tiles.
constexpr int kWaves = 4;               // waves per workgroup
constexpr int kPairCols = 32;           // columns of a tile pair
constexpr int kMaxSlices = 16;          // ordered partial sums per k-split, at most
constexpr int kPairsS = kWaves;         // tile pairs per workgroup, staged path
constexpr int kMaxMTiles = 9;           // up to 144 rows per forward pass
constexpr int kMaxRows = kMaxMTiles * 16;
constexpr int kDirectMT = 2;            // row tiles of the direct path (up to 32 rows)
constexpr int kStepRows = kDirectMT * 16;  // rows of a persistent-kernel pass
constexpr int kAttnBlock = 64;          // keys per attention block (absolute positions)
constexpr int kAttnSpan = 2;            // blocks per attention span (the first merge level)
constexpr int kAttnSpanKeys = kAttnSpan * kAttnBlock;
constexpr int kMaxSplits = 16;          // largest k-split count of a GEMM
constexpr int kMaxUnits = 24;           // (pair, split) units per workgroup, balanced direct path
constexpr int kMaxBlocks = 512;         // attention blocks per row (positions < 32768)

// Column order of a packed matrix (pack_kernel): which matrix row (output
// column) sits at column 16 j + c of tile pair tp.
enum PackMap {
  PACK_IDENTITY = 0,   // n = 32 tp + 16 j + c
  PACK_GATE_UP = 1,    // rows [gate; up] (F each): n = j F + 16 tp + c
  PACK_ROPE_PAIRS = 2  // heads of d rows: dims i and i + d/2 share a pair
};

// One processed row of a forward pass.
struct RowDesc {
  int32_t token;   // embedding row, or -1: take audio staging row `src`
  int32_t src;     // audio staging row
  int32_t pos;     // position (also the KV cache row it writes)
  int32_t slot;    // KV cache slot of its request
  int32_t cmp;     // candidate its greedy token is compared with (-1: none)
  int32_t pad[3];
};

// One request of a forward pass: rows [row_start, row_start + W).
struct ReqDesc {
  int32_t row_start, W, L0, slot;
};

struct StepOut {
  int32_t accepted, correction, nan_flag, pad;
};

enum AMode { A_PLAIN = 0, A_NORM = 1 };
// EPI_DOWN is EPI_RESID under its own id: the O and down projections then
// run as distinct kernel instantiations, so profiles attribute them apart.
enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_ARGMAX = 3, EPI_DOWN = 4 };

struct GemmArgs {
  const uint4* W;        // packed weight tiles
  int N, K, KT, KS, ktps;
  int np;                // tile pairs per workgroup on the direct path (1 or 2)
  int ns;                // ordered slices per k-split (4 or 16)
  int G;                 // balanced direct path: workgroups sharing the units (0: one unit
                         // group per workgroup)
  int M, MT;
  int rg_grid;           // staged path with row groups: row groups of 3, 2 tiles are
                         // used only if their grid reaches rg_grid workgroups (else 1 tile)
  // A operand: activation planes [kMaxRows][K].  For A_NORM the planes
  // hold x * g (residual times RMSNorm gain) and the epilogue multiplies
  // row m by 1 / sqrt(sum(x^2) / K + eps) from the sum-of-squares partials.
  const void* A;
  long long a_plane;
  const float* sumsq;    // A_NORM: per-pair partials [kMaxRows][K / 32]
  int n_norm_pairs;
  float eps;
  // split-K scratch
  float* part;           // [KS][M][N]
  int* counters;         // one per workgroup tile, zero between launches
  // epilogue
  const RowDesc* rows;
  const float* bias;     // EPI_QKV (may be null)
  float* q_out;          // EPI_QKV: [M][n_q*d]
  float* k_cache;        // EPI_QKV: this layer's K cache (layout: AttnArgs), slot stride `slot_stride`
  float* v_cache;
  long long slot_stride; // float32 units between slots
  int kv_cap;            // positions per head (a multiple of 64)
  int n_q, n_kv, head_dim;
  const float* rope_cs;  // [kv_cap][head_dim/2][2] (cos, sin)
  const float* x;        // EPI_RESID: residual [M][N] read
  float* x_out;          // EPI_RESID: x + Y written (may equal x)
  float* sumsq_out;      // EPI_RESID: per-pair partials [kMaxRows][N / 32]
  const float* gain_next;// EPI_RESID: RMSNorm gain of the next consumer of x
  void* out;             // EPI_RESID: planes of x * gain_next; EPI_SWIGLU: planes of h
  long long out_plane;
  float* logits;         // EPI_ARGMAX: optional [M][N]
  float* amax_val;       // EPI_ARGMAX: per-pair partials [kMaxRows][N / 32]: largest value,
  float* amax_val2;      //   second-largest value,
  int* amax_idx;         //   lowest column holding the largest value
};

// KV cache of one layer and slot, per KV head (kv_cap * d float32 units
// each for K and for V):
//   K, bf16 models: [pos][2][d] bf16, the (hi, lo) pair of each value, hi
//   row then lo row per position; float32 models: [pos][d] float32.
//   V: blocks of 32 positions; block pos / 32 holds [parts][d][32] elements
//   (v_elem), so that the values of one 32-key chunk are one contiguous
//   run of d x 128 bytes: bf16 models hold the hi plane then
//   the lo plane, the keys of the block reordered (v_col) so that the eight
//   keys one lane group multiplies in p v are adjacent; float32 models hold
//   one float32 plane in key order.
// hi = bf16(x) and lo = bf16(x - hi): the operands of the attention's
// matrix-core products, stored once when the row is appended.
//
// v_col: within a group of 32, key 16 t + 4 g + e (t < 2, g < 4, e < 4)
// sits at 8 g + 4 t + e.
__host__ __device__ inline int v_col(int pos) {
  return (pos & ~31) | (((pos >> 2) & 3) << 3) | (((pos >> 4) & 1) << 2) | (pos & 3);
}
// Element index (bf16 or float32 units) of V value (pos, part, dimension
// dd) of one KV head with d dimensions.
__host__ __device__ inline size_t v_elem(int pos, int part, int dd, int d, bool bf16) {
  const int parts = bf16 ? 2 : 1;
  const int col = bf16 ? (v_col(pos) & 31) : (pos & 31);
  return ((size_t)(pos >> 5) * parts + part) * d * 32 + (size_t)dd * 32 + col;
}

struct AttnArgs {
  const float* q;        // [M][n_q*d]
  const float* k_cache;  // this layer
  const float* v_cache;
  long long slot_stride; // float32 units between slots
  int kv_cap;            // positions per head (a multiple of 64)
  const RowDesc* rows;
  const ReqDesc* reqs;
  int n_q, n_kv, head_dim;
  float scale;           // log2(e) / sqrt(head_dim): scores in base-2 units
  float* pacc;           // span states [row][n_q][part_spans][d]
  float* pml;            // [row][n_q][part_spans][2]: running maximum and sum
  int part_spans;        // spans per (row, head) in the state arrays
  int* attn_cnt;         // merge_last: finished spans per (request, KV head, row block), zero between
                         // launches; [request][KV head][2 n_q / n_kv]: a request has at most 32 rows
                         // (max_k <= 31), so a KV head's rows fill at most that many 16-row blocks
  int merge_last;        // 1: the last item of a block merges its rows (no merge kernel)
  void* out;             // planes [kMaxRows][n_q*d]
  long long out_plane;
  int M;
  int attn_rt;           // row tiles per block of the verification kernel (0: chosen per launch)
  int cus;               // compute units the verification kernels may fill (the CU budget)
};

// Persistent step kernel (step.hip): one verification pass of up to 32 rows.
struct StepLayer {
  GemmArgs qkv, o, gu, down;
  AttnArgs attn;
};

struct StepArgs {
  const StepLayer* layers;   // device array, one per decoder layer
  int n_layers;
  GemmArgs lm;
  int M;                     // rows of the pass
  const RowDesc* rows;
  const void* embed;
  const void* audio;
  int hidden;
  const float* gain0;        // first RMSNorm gain
  float* x0;                 // embedding outputs (inputs of layer 0)
  float* sumsq0;
  void* xg0;
  long long xg0_plane;
  const ReqDesc* reqs;       // attention requests
  int n_reqs;
  int n_q, n_kv;
  const ReqDesc* fin_reqs;   // verified requests and their rows
  int n_fin;
  int fin_rows;
  int* row_tok;
  int* row_bad;
  float* row_margin;
  StepOut* out;
  int done_qkv, done_o, done_gu, done_down, done_lm;  // completion signals per GEMM phase
  int* phase_cnt;            // 3 + 6 * n_layers counters, cleared by the launcher
  int* err;                  // set when a wait times out
  int spin_limit;
  long long* trace;          // optional [grid][3 + 6 * n_layers][3] wall-clock stamps
};

// Sets the launch attributes of kernels that may use more than 64 KiB of
// LDS; call once per process before the first launch (prepare_kernels
// calls prepare_step_kernels).
hipError_t prepare_kernels();
// The host-side conditions of the balanced path (gemm_range_direct):
// 1 <= G <= units, at most kMaxUnits units per workgroup, every split at
// least kWaves k-steps, KS <= kMaxSplits, kWaves slices, MT <= kDirectMT.
bool range_plan_ok(const GemmArgs& a);
hipError_t prepare_step_kernels();

// Launchers (all asynchronous on `s`).  `bf16` selects the model dtype.
// map: PackMap; arg: F for PACK_GATE_UP, the head dimension for PACK_ROPE_PAIRS.
hipError_t launch_pack(bool bf16, const void* src, uint4* dst, int N, int K, int map, int arg,
                       hipStream_t s);
hipError_t launch_embed(bool bf16, const RowDesc* rows, int M, const void* embed, const void* audio,
                        int H, const float* gain, float* x, float* sumsq, void* xg, long long xg_plane,
                        hipStream_t s);
hipError_t launch_gemm(bool bf16, int amode, int epi, const GemmArgs& a, hipStream_t s);
int step_lds_bytes(int MT, int head_dim, int hidden);
// Slice length of the register-resident balanced variant for a gate/up
// plan (KS, KT) with one row tile, or 0: the persistent kernel to launch.
int step_ra_slice(bool bf16, int KS, int KT);
hipError_t step_occupancy(bool bf16, int MT, int head_dim, int hidden, int sl, int* blocks_per_cu);
hipError_t launch_step(bool bf16, int MT, int head_dim, int sl, const StepArgs& a, int grid, int n_counters,
                       hipStream_t s);
// Attention over n_reqs requests (attn.h).  Verification passes (rows of a
// request <= 32): max_blocks bounds the 64-key blocks of any request and
// sizes the grid (any value covers every cache length; the grid is at most
// kAttnGrid workgroups).  prefill: one request of up to kMaxRows rows.
hipError_t launch_attention(bool bf16, const AttnArgs& a, int n_reqs, int max_blocks, bool prefill, hipStream_t s);
// n_rows = sum of the requests' W; counters: one per request, zero between launches.
// Writes each verified row's greedy token, non-finite flag and top-2 margin.
hipError_t launch_finish(const RowDesc* rows, const ReqDesc* reqs, int n_reqs, int n_rows,
                         const float* amax_val, const float* amax_val2, const int* amax_idx, int n_pairs,
                         int* row_tok, int* row_bad, float* row_margin, int* counters, StepOut* out,
                         hipStream_t s);

// Zeroes n ints (a kernel, not a memset, so that it may be captured).
hipError_t launch_fill_zero(int* p, int n, hipStream_t s);

// The library's static scratch array (static_scratch.hip) on the current
// device: its device address (looked up once per device) and size.
hipError_t static_scratch(void** ptr, size_t* bytes);

// Streams n16 16-byte units of buf with `grid` workgroups (read-bandwidth
// reference); n16 must split into whole 8 KiB runs per wave.
hipError_t launch_stream_read(const uint4* buf, long long n16, int grid, unsigned* out, hipStream_t s);

}  // namespace as2d
