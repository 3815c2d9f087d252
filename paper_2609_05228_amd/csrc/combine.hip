// Gate-weighted combine of the sparsified MoE output (Eq. ace_sparse_output):
//   y_t = sum_{i in I_t} ghat_{t,i} Y[slot_row[t,i]]  (+ the shared expert's row)
// where Y rows are either bf16/fp32 rows or, after a K-split small-batch down
// GEMM, the fp32 sum of their partials (added in split order).  Slots are added
// in slot order with fp32 FMA: deterministic, no atomics.
//  * rows: one workgroup per token, 16-byte vectors across the hidden dimension;
//    every kept slot's vector is loaded before the first FMA, so the loads of a
//    token are in flight together;
//  * K-split partials (small batches): one workgroup per (128-column block,
//    token); thread (slot i, 4 columns) sums slot i's partials in split order
//    with every load in flight at once, then one thread per 4 columns adds the
//    slots in slot order.
#include "ace_internal.h"

namespace ace {

namespace {

template <typename T> struct V;
template <> struct V<bf16_t> {
  static constexpr int n = 8;
  typedef uint4 raw;
  static __device__ __forceinline__ raw load(const bf16_t *p) { return *reinterpret_cast<const uint4 *>(p); }
  static __device__ __forceinline__ void cvt(const raw &q, float v[8]) {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(w[j] << 16);
      v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
    }
  }
  static __device__ __forceinline__ void store(bf16_t *p, const float v[8]) {
    *reinterpret_cast<uint4 *>(p) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                               pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
  }
  static __device__ __forceinline__ void store4(bf16_t *p, const float v[4]) {
    *reinterpret_cast<uint2 *>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
  static __device__ __forceinline__ void load4(const bf16_t *p, float v[4]) {
    const uint2 q = *reinterpret_cast<const uint2 *>(p);
    v[0] = __uint_as_float(q.x << 16);
    v[1] = __uint_as_float(q.x & 0xFFFF0000u);
    v[2] = __uint_as_float(q.y << 16);
    v[3] = __uint_as_float(q.y & 0xFFFF0000u);
  }
};
template <> struct V<float> {
  static constexpr int n = 4;
  typedef float4 raw;
  static __device__ __forceinline__ raw load(const float *p) { return *reinterpret_cast<const float4 *>(p); }
  static __device__ __forceinline__ void cvt(const raw &q, float v[4]) {
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  }
  static __device__ __forceinline__ void store(float *p, const float v[4]) {
    *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
  static __device__ __forceinline__ void store4(float *p, const float v[4]) { store(p, v); }
  static __device__ __forceinline__ void load4(const float *p, float v[4]) { cvt(load(p), v); }
};

template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  constexpr int VN = V<T>::n;
  __shared__ int rows[kMaxK];
  __shared__ float gs[kMaxK];
  const int t = blockIdx.x;
  if (threadIdx.x < kMaxK) {
    const bool in = static_cast<int>(threadIdx.x) < a.k;
    rows[threadIdx.x] = in ? a.slot_row[static_cast<size_t>(t) * a.k + threadIdx.x] : -1;
    gs[threadIdx.x] = in ? a.gates[static_cast<size_t>(t) * a.k + threadIdx.x] : 0.f;
  }
  __syncthreads();
  const T *Y = static_cast<const T *>(a.Y);
  const T *Ys = static_cast<const T *>(a.Ys);
  T *y = static_cast<T *>(a.y);
  for (int c = threadIdx.x * VN; c < a.d; c += 256 * VN) {
    typename V<T>::raw q[kMaxK];
#pragma unroll
    for (int i = 0; i < kMaxK; ++i)
      if (rows[i] >= 0) q[i] = V<T>::load(Y + static_cast<size_t>(rows[i]) * a.d + c);
    typename V<T>::raw qs;
    if (Ys) qs = V<T>::load(Ys + static_cast<size_t>(t) * a.d + c);
    float acc[VN];
#pragma unroll
    for (int j = 0; j < VN; ++j) acc[j] = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      if (rows[i] < 0) continue;
      float v[VN];
      V<T>::cvt(q[i], v);
      const float g = gs[i];
#pragma unroll
      for (int j = 0; j < VN; ++j) acc[j] = fmaf(g, v[j], acc[j]);
    }
    if (Ys) {
      float v[VN];
      V<T>::cvt(qs, v);
#pragma unroll
      for (int j = 0; j < VN; ++j) acc[j] += v[j];
    }
    V<T>::store(y + static_cast<size_t>(t) * a.d + c, acc);
  }
}

constexpr int kSplitCols = 128;  // columns of one split-combine workgroup
constexpr int kMaxSplits = 8;    // K splits of the small-batch down GEMM

template <typename T>
__global__ __launch_bounds__(256) void combine_split_kernel(CombineArgs a) {
  __shared__ float vs[kMaxK][kSplitCols + 4];
  __shared__ int rows[kMaxK];
  __shared__ float gs[kMaxK];
  const int t = blockIdx.y;
  const int tid = threadIdx.x;
  if (tid < kMaxK) {
    const bool in = tid < a.k;
    rows[tid] = in ? a.slot_row[static_cast<size_t>(t) * a.k + tid] : -1;
    gs[tid] = in ? a.gates[static_cast<size_t>(t) * a.k + tid] : 0.f;
  }
  __syncthreads();
  const int i = tid >> 5, cg = tid & 31;  // slot, 4-column group
  const int c = blockIdx.x * kSplitCols + 4 * cg;
  const int r = rows[i];
  if (r >= 0) {
    float4 q[kMaxSplits];
#pragma unroll
    for (int s = 0; s < kMaxSplits; ++s)
      if (s < a.ysplits) q[s] = *reinterpret_cast<const float4 *>(a.Ypart + (static_cast<size_t>(s) * a.rows_cap + r) * a.d + c);
    float v[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kMaxSplits; ++s) {
      if (s >= a.ysplits) break;
      v[0] += q[s].x;
      v[1] += q[s].y;
      v[2] += q[s].z;
      v[3] += q[s].w;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) vs[i][4 * cg + j] = v[j];
  }
  __syncthreads();
  if (tid < 32) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kMaxK; ++s) {
      if (rows[s] < 0) continue;
      const float g = gs[s];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fmaf(g, vs[s][4 * tid + j], acc[j]);
    }
    if (a.Ys) {
      float v[4];
      V<T>::load4(static_cast<const T *>(a.Ys) + static_cast<size_t>(t) * a.d + c, v);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] += v[j];
    }
    V<T>::store4(static_cast<T *>(a.y) + static_cast<size_t>(t) * a.d + c, acc);
  }
}

}  // namespace

hipError_t launch_combine(const CombineArgs &a, bool bf16, hipStream_t stream) {
  if (a.T <= 0) return hipSuccess;
  if (a.Ypart) {
    if (a.ysplits < 1 || a.ysplits > kMaxSplits || a.d % kSplitCols != 0) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(a.d / kSplitCols), static_cast<unsigned>(a.T));
    if (bf16)
      combine_split_kernel<bf16_t><<<grid, 256, 0, stream>>>(a);
    else
      combine_split_kernel<float><<<grid, 256, 0, stream>>>(a);
  } else if (bf16) {
    combine_kernel<bf16_t><<<dim3(a.T), 256, 0, stream>>>(a);
  } else {
    combine_kernel<float><<<dim3(a.T), 256, 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace ace
