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
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
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

constexpr int kMaxN = 256;   // routed experts supported by the router kernel
constexpr int kMaxK = 8;     // top-k supported by the router kernel
constexpr int kTileM = 256;  // rows of one grouped-GEMM M tile (the dispatch plan's tile size)
constexpr int kRouteTokens = 16;  // tokens per router workgroup (one dispatch-plan chunk)

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
  int T, d, N, k, m_min;
  float tau, eps, rms_eps;
  int skip_disable;
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
  int dense_rows;         // > 0: dense single-group mode with this many rows
  int max_groups;         // upper bound of M tiles (grid sizing)
  int d, m;               // hidden and intermediate sizes of this GEMM's expert(s)
};

struct CombineArgs {
  const void *Y;          // [rows, d] routed expert outputs in compacted order
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

}  // namespace ace
