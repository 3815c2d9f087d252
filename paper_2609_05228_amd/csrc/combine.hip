// Gate-weighted combine of the sparsified MoE output (Eq. ace_sparse_output):
//   y_t = sum_{i in I_t} ghat_{t,i} Y[slot_row[t,i]]  (+ the shared expert's row)
// where Y rows are either bf16/fp32 rows or, after a K-split small-batch down
// GEMM, the fp32 sum of their partials (added in split order).
// One workgroup per token, 16-byte vectors across the hidden dimension, slots
// added in slot order with fp32 FMA: deterministic, no atomics.
#include "ace_internal.h"

namespace ace {

namespace {

template <typename T> struct V;
template <> struct V<bf16_t> {
  static constexpr int n = 8;
  static __device__ __forceinline__ void load(const bf16_t *p, float v[8]) {
    const uint4 q = *reinterpret_cast<const uint4 *>(p);
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
};
template <> struct V<float> {
  static constexpr int n = 4;
  static __device__ __forceinline__ void load(const float *p, float v[4]) {
    const float4 q = *reinterpret_cast<const float4 *>(p);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  }
  static __device__ __forceinline__ void store(float *p, const float v[4]) {
    *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};

template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  constexpr int VN = V<T>::n;
  __shared__ int rows[kMaxK];
  __shared__ float gs[kMaxK];
  const int t = blockIdx.x;
  if (threadIdx.x < a.k) {
    rows[threadIdx.x] = a.slot_row[static_cast<size_t>(t) * a.k + threadIdx.x];
    gs[threadIdx.x] = a.gates[static_cast<size_t>(t) * a.k + threadIdx.x];
  }
  __syncthreads();
  const T *Y = static_cast<const T *>(a.Y);
  const T *Ys = static_cast<const T *>(a.Ys);
  T *y = static_cast<T *>(a.y);
  for (int c = threadIdx.x * VN; c < a.d; c += 256 * VN) {
    float acc[VN];
#pragma unroll
    for (int j = 0; j < VN; ++j) acc[j] = 0.f;
    for (int i = 0; i < a.k; ++i) {
      const int r = rows[i];
      if (r < 0) continue;
      float v[VN];
      if (a.Ypart) {
        // K-split partial sums of this row, added in split order
#pragma unroll
        for (int j = 0; j < VN; ++j) v[j] = 0.f;
        for (int s = 0; s < a.ysplits; ++s) {
          const float *p = a.Ypart + (static_cast<size_t>(s) * a.rows_cap + r) * a.d + c;
#pragma unroll
          for (int j = 0; j < VN; j += 4) {
            const float4 q = *reinterpret_cast<const float4 *>(p + j);
            v[j] += q.x;
            v[j + 1] += q.y;
            v[j + 2] += q.z;
            v[j + 3] += q.w;
          }
        }
      } else {
        V<T>::load(Y + static_cast<size_t>(r) * a.d + c, v);
      }
      const float g = gs[i];
#pragma unroll
      for (int j = 0; j < VN; ++j) acc[j] = fmaf(g, v[j], acc[j]);
    }
    if (Ys) {
      float v[VN];
      V<T>::load(Ys + static_cast<size_t>(t) * a.d + c, v);
#pragma unroll
      for (int j = 0; j < VN; ++j) acc[j] += v[j];
    }
    V<T>::store(y + static_cast<size_t>(t) * a.d + c, acc);
  }
}

}  // namespace

hipError_t launch_combine(const CombineArgs &a, bool bf16, hipStream_t stream) {
  if (a.T <= 0) return hipSuccess;
  if (bf16)
    combine_kernel<bf16_t><<<dim3(a.T), 256, 0, stream>>>(a);
  else
    combine_kernel<float><<<dim3(a.T), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
