// Internal declarations shared by the ACE HIP kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ace {

// ---------------------------------------------------------------- element types
typedef uint16_t bf16_t;  // bfloat16 bit pattern

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// round to nearest, ties to even (inputs here are finite)
typedef __bf16 bf16x2_hw_t __attribute__((ext_vector_type(2)));
typedef float f32x2_hw_t __attribute__((ext_vector_type(2)));

// two fp32 -> two bf16 packed in one dword (lo in bits 0-15), round to
// nearest even, one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_hw_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_hw_t));
}

__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return static_cast<bf16_t>(pack_bf16x2(f, 0.f) & 0xFFFFu);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float *p) { return *p; }
  static __device__ __forceinline__ float to_f32(float v) { return v; }
  static __device__ __forceinline__ float from_f32(float v) { return v; }
};
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t *p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ float to_f32(bf16_t v) { return bf16_to_f32(v); }
  static __device__ __forceinline__ bf16_t from_f32(float v) { return f32_to_bf16(v); }
};

// SiLU of a value whose product with the up projection is rounded to bf16 right
// after: the hardware base-2 exponential and reciprocal (each about 1 ulp of
// fp32, far below bf16's 8-bit significand) instead of an exact division.
// v -> -inf gives -0, v -> +inf gives v.  fp32 layers keep the exact form.
__device__ __forceinline__ float silu_for_bf16(float v) {
  const float e = __builtin_amdgcn_exp2f(v * -1.4426950408889634f);  // exp(-v)
  return v * __builtin_amdgcn_rcpf(1.0f + e);
}

constexpr int kMaxN = 256;   // routed experts supported by the router kernel
constexpr int kMaxK = 8;     // top-k supported by the router kernel
constexpr int kTileM = 256;  // rows of one grouped-GEMM M tile (the dispatch plan's tile size)
constexpr int kRouteTokens = 16;  // tokens per router workgroup (one dispatch-plan chunk)
constexpr int kRouteMaxSlices = 16;  // K slices of the small-batch router
constexpr int kRoutePairMinChunks = 256;  // bf16 batches of more chunks: one router workgroup per chunk pair
constexpr int kRouteMaxSplitChunks = 16;  // most chunks that take the small-batch (K-slice) router path

// 16-expert tiles the router kernels are compiled for: 1, 2, 4, 8 or 16 (>= N / 16)
inline int route_expert_tiles(int N) {
  const int need = (N + 15) / 16;
  return need <= 1 ? 1 : need <= 2 ? 2 : need <= 4 ? 4 : need <= 8 ? 8 : 16;
}

// ---------------------------------------------------------------- kernel arguments
struct RouteArgs {
  const void *x;          // [T, d]
  const void *gamma;      // [d]
  const void *w_router;   // [N, d]
  const float *b_router;  // [N] or null
  const float *a_gsp;     // [N]
  const float *a_rcr;     // [N]
  void *xn;               // [T, d] normalised input (expert GEMM operand)
  int32_t *topk_idx;      // [T, k]
  uint8_t *keep;          // [T, k]
  float *gates;           // [T, k] ghat
  float *scores;          // [T, k] c, or null
  int32_t *slot_row;      // [T, k]: -1 for skipped slots (kept slots are filled by the plan)
  uint8_t *local_rank;    // [T, k]: rank of a kept slot among its chunk's kept slots of that expert
  uint8_t *chunk_count;   // [G, N]: kept slots per (16-token chunk, expert)
  float *zpart;           // [ksplit, T, zstride]: partial logits of the K slices (ksplit > 0)
  float *sspart;          // [ksplit, T]: partial sums of squares of x
  int ksplit;             // 0: one fused kernel; else K slices (<= 16, dividing d / 32)
  // one chunk (T <= 16): the select workgroup also writes the dispatch plan
  int32_t *counts;        // [N]
  int32_t *offsets;       // [N+1]
  int32_t *perm;          // [T*k]
  int32_t *tile_expert, *tile_row0, *tile_rows, *n_tiles;
  int zstride;            // 16 * route_expert_tiles(N)
  int T, d, N, k, m_min;
  float tau, eps, rms_eps;
  int skip_disable;
  int fusion;             // ace_fusion: contribution rule (ACE: max)
};

struct PlanArgs {
  const uint8_t *chunk_count;        // [G, N]
  const uint8_t *local_rank;         // [T, k]
  const int32_t *topk_idx;           // [T, k]
  const uint8_t *keep;               // [T, k]
  int32_t *chunk_base;               // [N, G]: kept slots of expert e in chunks before g
  int32_t *counts;                   // [N]
  int32_t *offsets;                  // [N+1]
  int32_t *perm;                     // [T*k]
  int32_t *slot_row;                 // [T, k]
  int32_t *tile_expert;              // [max_tiles]
  int32_t *tile_row0;                // [max_tiles]
  int32_t *tile_rows;                // [max_tiles]
  int32_t *n_tiles;                  // [1]
  int32_t *tile_order;               // [max_tiles] or null: the gate/up launch's tile order (see plan_kernel)
  int T, k, N, G;
};

// Grouped GEMM over the dispatch plan.  Tile g covers rows tile_row0[g] ..
// tile_row0[g] + tile_rows[g] - 1 of the compacted slot order, all routed to
// expert tile_expert[g].  In dense mode (dense_rows > 0) tile g covers rows
// g*kTileM .. of a single group with identity row->token map and expert 0.
struct GemmArgs {
  const void *act;        // gate/up: xn [T, d] (gathered through perm); down: H [rows, m]
  const int32_t *perm;    // row -> token (gate/up, routed); null in dense mode / for down
  const void *w0;         // gate/up: w_gate [E, m, d]; down: w_down [E, d, m]
  const void *w1;         // gate/up: w_up   [E, m, d]; down: unused
  void *out;              // gate/up: H [rows, m]; down: Y [rows, d]
  const int32_t *tile_expert, *tile_row0, *tile_rows, *n_tiles;
  const int32_t *tile_order;  // null: tiles in list order; else grid tile g is list tile tile_order[g]
  int dense_rows;         // > 0: dense single-group mode with this many rows
  int max_groups;         // upper bound of M tiles (grid sizing)
  int d, m;               // hidden and intermediate sizes of this GEMM's expert(s)
  // A dense expert appended to the routed tiles (bf16 grouped GEMM): tiles
  // n_tiles[0] .. n_tiles[0] + sh_tiles - 1 cover its rows (t - n_tiles[0]) * kTileM ..
  // with the identity row map, its own operands and its own output.  0: none.
  int sh_tiles, sh_rows;
  const void *sh_act, *sh_w0, *sh_w1;
  void *sh_out;
};

// Small-batch (decode) grouped GEMM: the same tiles, split over K into
// `splits` parts when the batch is too small to fill the GPU otherwise.
struct SkinnyArgs {
  GemmArgs g;
  int splits;      // K splits (1: write H / Y in bf16 directly)
  int rows_cap;    // row capacity of a partial-sum plane (T * k)
  float *part0;    // gate/up: gate partials [splits, rows_cap, m]; down: Y partials [splits, rows_cap, d]
  float *part1;    // gate/up: up partials [splits, rows_cap, m]
  // self_plan (routed gate/up, 2-4 router chunks): each wave derives its tile (the
  // grp-th expert with kept slots) and the tokens of its rows from the router's
  // per-chunk counts and the routing, instead of reading a plan; one item per
  // tile writes its slots' rows (slot_row, perm), item 0 writes counts, offsets
  // and the tile list (into the buffers g's tile pointers name) that the down
  // kernel reads
  bool self_plan;
  const int32_t *topk_idx;     // [T, k]
  const uint8_t *keep;         // [T, k]
  const uint8_t *chunk_count;  // [G, N]
  int32_t *counts, *offsets, *perm, *slot_row;
  int32_t *tile_expert, *tile_row0, *tile_rows, *n_tiles;
  int T, k, N, G;
};

struct CombineArgs {
  const void *Y;          // [rows, d] routed expert outputs in compacted order, or null
  const float *Ypart;     // [ysplits, rows_cap, d] fp32 partial sums of Y, or null
  int ysplits, rows_cap;
  const void *Ys;         // [T, d] shared-expert output, or null
  const int32_t *slot_row;  // [T, k]
  const float *gates;       // [T, k]
  void *y;                // [T, d]
  int T, d, k;
};

// ---------------------------------------------------------------- launchers
// Each returns hipGetLastError() after enqueueing on `stream`.
hipError_t launch_route(const RouteArgs &a, bool bf16, hipStream_t stream);
hipError_t launch_plan(const PlanArgs &a, hipStream_t stream);
hipError_t launch_gateup(const GemmArgs &a, bool bf16, hipStream_t stream);
hipError_t launch_down(const GemmArgs &a, bool bf16, hipStream_t stream);
hipError_t launch_combine(const CombineArgs &a, bool bf16, hipStream_t stream);
// gate/up (gateup = true; reduces K-split partials into H when splits > 1, with
// n_rows = device count of rows in routed mode) or down
// whether launch_plan writes PlanArgs::tile_order for these sizes (the one-kernel plan)
bool plan_writes_order(const PlanArgs &a);
hipError_t launch_skinny(const SkinnyArgs &a, bool gateup, const int32_t *n_rows, hipStream_t stream);

// Offline GSP / RCR tables (Alg. 2, Alg. 3) in fp64
struct TablesCall {
  const void *gamma, *w_router, *w_gate, *w_up, *w_down;
  int N, d, m;
  double eps;
  bool bf16;
  void *workspace;  // tables_workspace_bytes(N, d, m)
  float *a_gsp, *a_rcr;
  double *a_gsp64, *a_rcr64;  // optional
};
size_t tables_workspace_bytes(int N, int d, int m);
hipError_t launch_tables(const TablesCall &c, hipStream_t stream);

// App. C.1 threshold mapping: up to kTauMaxQ budgets per call; workspace of tau_workspace_bytes()
constexpr int kTauMaxQ = 8;
size_t tau_workspace_bytes();
hipError_t launch_tau_map(const float *scores, long long n_rows, int k, int m_min, const double *q, int n_q,
                          float *tau, long long *m_q_out, long long *n_cand_out, void *workspace,
                          hipStream_t stream);

}  // namespace ace
