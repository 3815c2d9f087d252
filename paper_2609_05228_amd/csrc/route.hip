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
//     sets (alternating 32-wide K blocks); the 8 partial sums per logit are added
//     in a fixed order, which keeps the accumulated rounding near 2e-7 for
//     d = 2048.  The same pass writes x_in, rounded to the GEMM dtype, for the
//     expert GEMMs.
//     The hidden dimension is walked in 32-wide blocks (16-byte loads per lane)
//     with the next block's operands loaded before the current block's MFMAs.
//  3. Each 16-lane group of a wave takes one token (4 tokens per wave at once):
//     top-k by k rounds of a 16-lane arg-max (ties go to the lower expert id),
//     gates g = exp(z_i - z_1) / sum_j exp(z_j - z_1) over the k selected logits
//     (the softmax over all N experts cancels in the renormalised gate), then
//     Alg. 4 evaluated redundantly in every lane of the group (k <= 8 scalars),
//     and lane i < k of the group writes slot i.
//  4. For the dispatch plan, each kept slot gets its rank among this
//     workgroup's kept slots of the same expert in token order (from a 16-bit
//     token mask per expert in LDS), and the workgroup writes its per-expert
//     kept counts.  No global atomics: the plan is independent of scheduling.
#include "ace_internal.h"

namespace ace {

namespace {

constexpr int kTok = kRouteTokens;  // tokens per workgroup

// 8 consecutive elements: raw storage and conversion
template <typename T> struct Oct;
template <> struct Oct<float> {
  struct raw {
    float4 lo, hi;
  };
  static __device__ __forceinline__ raw load(const float *p) {
    raw r;
    r.lo = *reinterpret_cast<const float4 *>(p);
    r.hi = *reinterpret_cast<const float4 *>(p + 4);
    return r;
  }
  static __device__ __forceinline__ void cvt(const raw &q, float v[8]) {
    v[0] = q.lo.x; v[1] = q.lo.y; v[2] = q.lo.z; v[3] = q.lo.w;
    v[4] = q.hi.x; v[5] = q.hi.y; v[6] = q.hi.z; v[7] = q.hi.w;
  }
  static __device__ __forceinline__ void store(float *p, const float v[8]) {
    *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4 *>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
};
template <> struct Oct<bf16_t> {
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
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w[j] = static_cast<uint32_t>(f32_to_bf16(v[2 * j])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * j + 1])) << 16);
    *reinterpret_cast<uint4 *>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

template <typename T>
__device__ __forceinline__ void load4(const T *p, float v[4]);
template <>
__device__ __forceinline__ void load4<float>(const float *p, float v[4]) {
  const float4 q = *reinterpret_cast<const float4 *>(p);
  v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
}
template <>
__device__ __forceinline__ void load4<bf16_t>(const bf16_t *p, float v[4]) {
  const uint2 q = *reinterpret_cast<const uint2 *>(p);
  v[0] = __uint_as_float(q.x << 16);
  v[1] = __uint_as_float(q.x & 0xFFFF0000u);
  v[2] = __uint_as_float(q.y << 16);
  v[3] = __uint_as_float(q.y & 0xFFFF0000u);
}

__device__ __forceinline__ bool better(float v, int e, float bv, int be) {
  return v > bv || (v == bv && e < be);
}

// Operands of one 32-wide K block for one lane: the lane's 8 consecutive k of
// its token row, of gamma and of NT router rows.  MFMA j of the block takes
// element j from every lane, so lane group g supplies k = kb + 8g + j to both
// operands and the block covers kb .. kb + 31.
template <typename T, int NT> struct Block {
  typename Oct<T>::raw x, g, w[NT];
};

template <typename T, int NT>
__device__ __forceinline__ void load_block(Block<T, NT> &b, const T *xrow, const T *gamma, const T *wr,
                                           int d, int N, int r16, int k) {
  b.x = Oct<T>::load(xrow + k);
  b.g = Oct<T>::load(gamma + k);
#pragma unroll
  for (int et = 0; et < NT; ++et) {
    const int e = min(et * 16 + r16, N - 1);  // rows past N reuse row N-1; their logits are never read
    b.w[et] = Oct<T>::load(wr + static_cast<size_t>(e) * d + k);
  }
}

template <typename T, int NT>
__device__ __forceinline__ void mfma_block(const Block<T, NT> &b, f32x4_t (&acc)[NT], float rs, bool tvalid,
                                           T *xnp) {
  float xv[8], gv[8], av[8];
  Oct<T>::cvt(b.x, xv);
  Oct<T>::cvt(b.g, gv);
#pragma unroll
  for (int j = 0; j < 8; ++j) av[j] = tvalid ? (xv[j] * rs) * gv[j] : 0.f;
  if (tvalid) Oct<T>::store(xnp, av);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int et = 0; et < NT; ++et) {
      float bv[8];
      Oct<T>::cvt(b.w[et], bv);
      acc[et] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j], bv[j], acc[et], 0, 0, 0);
    }
  }
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
  __shared__ uint32_t emask[NT * 16];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int t0 = blockIdx.x * kTok;
  const int d = a.d;
  const int N = a.N;
  for (int e = tid; e < NT * 16; e += 256) emask[e] = 0u;

  // ---- 1. RMS scale per token
  for (int j = 0; j < 4; ++j) {
    const int tl = wave * 4 + j;
    const int t = t0 + tl;
    float ss = 0.f;
    if (t < a.T) {
      const T *row = x + static_cast<size_t>(t) * d;
      for (int c = lane * 4; c < d; c += 256) {
        float v[4];
        load4<T>(row + c, v);
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

  // ---- 2. router logits on fp32 MFMA, two accumulator sets (even / odd K blocks)
  {
    const int r16 = lane & 15;  // A row (token) / B column (expert within a tile)
    const int grp = lane >> 4;  // K group of the MFMA operand
    const int t = t0 + r16;
    const bool tvalid = t < a.T;
    const float rs = rstd_s[r16];
    const int kq = d >> 2;         // this wave's K range, a multiple of 32
    const int nb = kq >> 5;        // 32-wide K blocks
    const int kbeg = wave * kq + grp * 8;
    const T *xrow = x + static_cast<size_t>(tvalid ? t : 0) * d;
    T *xnrow = xn + static_cast<size_t>(tvalid ? t : 0) * d;

    f32x4_t acc0[NT], acc1[NT];
#pragma unroll
    for (int et = 0; et < NT; ++et) {
      acc0[et] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      acc1[et] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    // the next block's operands are loaded before the current block's MFMAs
    Block<T, NT> b0, b1;
    load_block<T, NT>(b0, xrow, gamma, wr, d, N, r16, kbeg);
    int j = 0;
    for (; j + 1 < nb; j += 2) {
      const int k = kbeg + 32 * j;
      load_block<T, NT>(b1, xrow, gamma, wr, d, N, r16, k + 32);
      mfma_block<T, NT>(b0, acc0, rs, tvalid, xnrow + k);
      load_block<T, NT>(b0, xrow, gamma, wr, d, N, r16, kbeg + 32 * min(j + 2, nb - 1));
      mfma_block<T, NT>(b1, acc1, rs, tvalid, xnrow + k + 32);
    }
    if (j < nb) mfma_block<T, NT>(b0, acc0, rs, tvalid, xnrow + kbeg + 32 * j);
    // D[row = token 4*grp + i][col = expert et*16 + r16]
#pragma unroll
    for (int et = 0; et < NT; ++et)
#pragma unroll
      for (int i = 0; i < 4; ++i) zp[wave][grp * 4 + i][et * 16 + r16] = acc0[et][i] + acc1[et][i];
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

  // ---- 3. top-k, gates and Alg. 4: one token per 16-lane group
  const int k = a.k;
  const int sub = lane & 15;
  const int tl = wave * 4 + (lane >> 4);
  const int t = t0 + tl;
  const bool tvalid = t < a.T;
  int my_e = -1;        // expert of this lane's slot (lane sub < k), -1 if none
  bool my_kept = false;
  {
    const float *zrow = zp[0][tl];
    float v[NT];
#pragma unroll
    for (int q = 0; q < NT; ++q) {
      const int e = sub + 16 * q;
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
        for (int q = 0; q < NT; ++q) {
          const int e = sub + 16 * q;
          if (e < N && !((taken >> q) & 1u) && better(v[q], e, bv, be)) {
            bv = v[q];
            be = e;
          }
        }
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) {
          const float ov = __shfl_xor(bv, off, 16);
          const int oe = __shfl_xor(be, off, 16);
          if (better(ov, oe, bv, be)) {
            bv = ov;
            be = oe;
          }
        }
        sel_e[i] = be;
        sel_z[i] = bv;
        if ((be & 15) == sub) taken |= 1u << (be >> 4);
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
      if (tvalid && i < k && i == sub) {
        const size_t o = static_cast<size_t>(t) * k + i;
        const float gh = a.skip_disable ? gsel[i] : (kept[i] ? gsel[i] / zgate : 0.f);
        a.topk_idx[o] = sel_e[i];
        a.keep[o] = kept[i] ? 1 : 0;
        a.gates[o] = gh;
        if (a.scores) a.scores[o] = c[i];
        if (!kept[i]) a.slot_row[o] = -1;
        my_e = sel_e[i];
        my_kept = kept[i];
      }
    }
  }
  // ---- 4. per-expert token masks of this workgroup -> local ranks and counts
  if (my_kept) atomicOr(&emask[my_e], 1u << tl);
  __syncthreads();
  if (my_kept) {
    const uint32_t below = emask[my_e] & ((1u << tl) - 1u);
    a.local_rank[static_cast<size_t>(t) * k + sub] = static_cast<uint8_t>(__popc(below));
  }
  for (int e = tid; e < N; e += 256)
    a.chunk_count[static_cast<size_t>(blockIdx.x) * N + e] = static_cast<uint8_t>(__popc(emask[e]));
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

}  // namespace

hipError_t launch_route(const RouteArgs &a, bool bf16, hipStream_t stream) {
  return bf16 ? launch_route_t<bf16_t>(a, stream) : launch_route_t<float>(a, stream);
}

}  // namespace ace
