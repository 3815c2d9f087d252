// Router and ACE skip mask: RMSNorm, router logits, softmax/top-k with gate
// renormalisation, and the per-token ACE skipping of Alg. 4 (dual-view scores,
// max fusion, top-1 and minimum-active safeguards, gate renormalisation).
//
// One workgroup (4 waves) owns 16 tokens.
//  1. Each wave computes the RMS scale of 4 tokens (fp32 sum of squares).
//  2. Router logits z = x_in W_r^T (App. B.2, Eq. app_router_logit) on fp32 MFMA
//     (v_mfma_f32_16x16x4f32): x_in is the un-rounded fp32 RMSNorm output, so the
//     top-k and skip decisions see fp32 logits, not bf16-rounded activations.
//     Wave w owns a quarter of the hidden dimension and keeps two accumulator
//     sets (alternating 16-wide K blocks); the 8 partial sums per logit are added
//     in a fixed order, which keeps the accumulated rounding near 2e-7 for
//     d = 2048.  The same pass writes x_in, rounded to the GEMM dtype, for the
//     expert GEMMs.
//  3. Each wave takes 4 tokens: top-k by k rounds of a wavefront arg-max (ties go
//     to the lower expert id), gates g = exp(z_i - z_1) / sum_j exp(z_j - z_1)
//     over the k selected logits (the softmax over all N experts cancels in the
//     renormalised gate), then Alg. 4 evaluated redundantly in every lane (k <= 8
//     scalars), and lane i < k writes slot i.  Kept (expert, token) pairs are
//     recorded in a per-expert token bitmap with integer atomic OR, which makes
//     the later dispatch order independent of scheduling.
#include "ace_internal.h"

namespace ace {

namespace {

constexpr int kTok = 16;  // tokens per workgroup

template <typename T> struct Vec4;
template <> struct Vec4<float> {
  static __device__ __forceinline__ void load(const float *p, float v[4]) {
    const float4 q = *reinterpret_cast<const float4 *>(p);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  }
  static __device__ __forceinline__ void store(float *p, const float v[4]) {
    *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct Vec4<bf16_t> {
  static __device__ __forceinline__ void load(const bf16_t *p, float v[4]) {
    const uint2 q = *reinterpret_cast<const uint2 *>(p);
    v[0] = __uint_as_float(q.x << 16);
    v[1] = __uint_as_float(q.x & 0xFFFF0000u);
    v[2] = __uint_as_float(q.y << 16);
    v[3] = __uint_as_float(q.y & 0xFFFF0000u);
  }
  static __device__ __forceinline__ void store(bf16_t *p, const float v[4]) {
    uint2 q;
    q.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
    q.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
    *reinterpret_cast<uint2 *>(p) = q;
  }
};

__device__ __forceinline__ bool better(float v, int e, float bv, int be) {
  return v > bv || (v == bv && e < be);
}

// NT = number of 16-expert tiles covered (N <= 16 * NT)
template <typename T, int NT>
__global__ __launch_bounds__(256) void route_kernel(RouteArgs a) {
  const T *__restrict__ x = static_cast<const T *>(a.x);
  const T *__restrict__ gamma = static_cast<const T *>(a.gamma);
  const T *__restrict__ wr = static_cast<const T *>(a.w_router);
  T *__restrict__ xn = static_cast<T *>(a.xn);

  __shared__ float rstd_s[kTok];
  __shared__ float zp[4][kTok][NT * 16 + 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int t0 = blockIdx.x * kTok;
  const int d = a.d;
  const int N = a.N;

  // ---- 1. RMS scale per token
  for (int j = 0; j < 4; ++j) {
    const int tl = wave * 4 + j;
    const int t = t0 + tl;
    float ss = 0.f;
    if (t < a.T) {
      const T *row = x + static_cast<size_t>(t) * d;
      for (int c = lane * 4; c < d; c += 256) {
        float v[4];
        Vec4<T>::load(row + c, v);
        ss = fmaf(v[0], v[0], ss);
        ss = fmaf(v[1], v[1], ss);
        ss = fmaf(v[2], v[2], ss);
        ss = fmaf(v[3], v[3], ss);
      }
    }
    for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
    if (lane == 0) rstd_s[tl] = (t < a.T) ? 1.0f / sqrtf(ss / static_cast<float>(d) + a.rms_eps) : 0.f;
  }
  __syncthreads();

  // ---- 2. router logits on fp32 MFMA
  {
    const int r16 = lane & 15;  // A row (token) / B column (expert within a tile)
    const int grp = lane >> 4;  // K group of the MFMA operand
    const int t = t0 + r16;
    const bool tvalid = t < a.T;
    const float rs = rstd_s[r16];
    const int kq = d >> 2;
    const int kbeg = wave * kq;
    const T *xrow = x + static_cast<size_t>(tvalid ? t : 0) * d;
    T *xnrow = xn + static_cast<size_t>(tvalid ? t : 0) * d;

    f32x4_t acc[2][NT];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int et = 0; et < NT; ++et) acc[s][et] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int kb = kbeg; kb < kbeg + kq; kb += 32) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int k = kb + s * 16 + grp * 4;
        float av[4] = {0.f, 0.f, 0.f, 0.f};
        if (tvalid) {
          float xv[4], gv[4];
          Vec4<T>::load(xrow + k, xv);
          Vec4<T>::load(gamma + k, gv);
#pragma unroll
          for (int j = 0; j < 4; ++j) av[j] = (xv[j] * rs) * gv[j];
          Vec4<T>::store(xnrow + k, av);
        }
#pragma unroll
        for (int et = 0; et < NT; ++et) {
          const int e = et * 16 + r16;
          float bv[4] = {0.f, 0.f, 0.f, 0.f};
          if (e < N) Vec4<T>::load(wr + static_cast<size_t>(e) * d + k, bv);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[s][et] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j], bv[j], acc[s][et], 0, 0, 0);
        }
      }
    }
    // D[row = token 4*grp + i][col = expert et*16 + r16]
#pragma unroll
    for (int et = 0; et < NT; ++et)
#pragma unroll
      for (int i = 0; i < 4; ++i) zp[wave][grp * 4 + i][et * 16 + r16] = acc[0][et][i] + acc[1][et][i];
  }
  __syncthreads();
  for (int idx = tid; idx < kTok * N; idx += 256) {
    const int tl = idx / N;
    const int e = idx - tl * N;
    float z = (zp[0][tl][e] + zp[1][tl][e]) + (zp[2][tl][e] + zp[3][tl][e]);
    if (a.b_router) z += a.b_router[e];
    zp[0][tl][e] = z;
  }
  __syncthreads();

  // ---- 3. top-k, gates and Alg. 4, one token at a time per wave
  const int k = a.k;
  for (int j = 0; j < 4; ++j) {
    const int tl = wave * 4 + j;
    const int t = t0 + tl;
    if (t >= a.T) break;
    const float *zrow = zp[0][tl];
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + 64 * q;
      v[q] = (e < N) ? zrow[e] : -INFINITY;
    }
    unsigned taken = 0;
    int sel_e[kMaxK];
    float sel_z[kMaxK];
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      sel_e[i] = 0;
      sel_z[i] = 0.f;
      if (i < k) {
        float bv = -INFINITY;
        int be = 0x7fffffff;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = lane + 64 * q;
          if (e < N && !((taken >> q) & 1u) && better(v[q], e, bv, be)) {
            bv = v[q];
            be = e;
          }
        }
        for (int off = 32; off > 0; off >>= 1) {
          const float ov = __shfl_xor(bv, off);
          const int oe = __shfl_xor(be, off);
          if (better(ov, oe, bv, be)) {
            bv = ov;
            be = oe;
          }
        }
        sel_e[i] = be;
        sel_z[i] = bv;
        if ((be & 63) == lane) taken |= 1u << (be >> 6);
      }
    }
    // renormalised top-k gates
    float gsel[kMaxK];
    float gsum = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      gsel[i] = (i < k) ? expf(sel_z[i] - sel_z[0]) : 0.f;
      gsum += gsel[i];
    }
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) gsel[i] = gsel[i] / gsum;

    // Alg. 4: s = g * A(e); p = s / (sum s + eps); c = max(p_GSP, p_RCR)
    float sg[kMaxK], sr[kMaxK];
    float zg = 0.f, zr = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      sg[i] = (i < k) ? gsel[i] * a.a_gsp[sel_e[i]] : 0.f;
      sr[i] = (i < k) ? gsel[i] * a.a_rcr[sel_e[i]] : 0.f;
      zg += sg[i];
      zr += sr[i];
    }
    zg += a.eps;
    zr += a.eps;
    float c[kMaxK];
    bool kept[kMaxK];
    int nkept = 0;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      const float pg = sg[i] / zg;
      const float pr = sr[i] / zr;
      c[i] = fmaxf(pg, pr);
      // skip only if both views are below tau; slot 0 is the top-1 expert
      const bool skip = !a.skip_disable && i > 0 && pg < a.tau && pr < a.tau;
      kept[i] = (i < k) && !skip;
      nkept += kept[i] ? 1 : 0;
    }
    if (!a.skip_disable && nkept < a.m_min) {
      // restore skipped slots by descending c (ties -> lower slot) up to m_min
      const int need = a.m_min - nkept;
      bool restore[kMaxK];
#pragma unroll
      for (int i = 0; i < kMaxK; ++i) {
        int rank = 0;
#pragma unroll
        for (int jj = 0; jj < kMaxK; ++jj)
          if (jj < k && !kept[jj] && jj != i && (c[jj] > c[i] || (c[jj] == c[i] && jj < i))) ++rank;
        restore[i] = (i < k) && !kept[i] && rank < need;
      }
#pragma unroll
      for (int i = 0; i < kMaxK; ++i) kept[i] = kept[i] || restore[i];
    }
    float zgate = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxK; ++i)
      if (kept[i]) zgate += gsel[i];
    zgate += a.eps;

#pragma unroll
    for (int i = 0; i < kMaxK; ++i) {
      if (i < k && i == lane) {
        const size_t o = static_cast<size_t>(t) * k + i;
        const float gh = a.skip_disable ? gsel[i] : (kept[i] ? gsel[i] / zgate : 0.f);
        a.topk_idx[o] = sel_e[i];
        a.keep[o] = kept[i] ? 1 : 0;
        a.gates[o] = gh;
        if (a.scores) a.scores[o] = c[i];
        if (kept[i]) {
          atomicOr(&a.bitmap[static_cast<size_t>(sel_e[i]) * a.W + (t >> 6)], 1ull << (t & 63));
        } else {
          a.slot_row[o] = -1;
        }
      }
    }
  }
}

template <typename T>
hipError_t launch_route_t(const RouteArgs &a, hipStream_t stream) {
  const dim3 grid((a.T + kTok - 1) / kTok);
  const int nt = (a.N + 15) / 16;
  if (nt <= 2)
    route_kernel<T, 2><<<grid, 256, 0, stream>>>(a);
  else if (nt <= 4)
    route_kernel<T, 4><<<grid, 256, 0, stream>>>(a);
  else if (nt <= 8)
    route_kernel<T, 8><<<grid, 256, 0, stream>>>(a);
  else
    route_kernel<T, 16><<<grid, 256, 0, stream>>>(a);
  return hipGetLastError();
}

__global__ void zero_u64_kernel(unsigned long long *p, size_t n) {
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<size_t>(gridDim.x) * blockDim.x)
    p[i] = 0ull;
}

}  // namespace

hipError_t launch_route(const RouteArgs &a, bool bf16, hipStream_t stream) {
  return bf16 ? launch_route_t<bf16_t>(a, stream) : launch_route_t<float>(a, stream);
}

hipError_t launch_zero_u64(unsigned long long *p, size_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  zero_u64_kernel<<<dim3(static_cast<unsigned>(blocks)), 256, 0, stream>>>(p, n);
  return hipGetLastError();
}

}  // namespace ace
