// Router and ACE skip mask: RMSNorm, router logits, softmax/top-k with gate
// renormalisation, and the per-token ACE skipping of Alg. 4 (dual-view scores,
// max fusion, top-1 and minimum-active safeguards, gate renormalisation).
//
// Per 16-token chunk (one dispatch-plan chunk):
//  1. Logits.  z[t][e] = rstd_t * sum_k (x[t,k] gamma[k]) W_r[e,k] + b[e]
//     (Sec. 3.1 x = x_bar Gamma; App. B.2, Eq. app_router_logit) with the RMS
//     scale factored out of the sum.  K is cut into 32-wide blocks; a wave
//     accumulates its blocks for 16 tokens x all N experts in MFMA
//     accumulators, plus the per-token sum of squares of x.
//       bf16: x and gamma are bf16, so x*gamma has at most 16 significant bits
//       and splits exactly into hi + lo, both bf16; the logits take two
//       v_mfma_f32_16x16x32_bf16 per 32 K (hi, then lo) against the bf16
//       router rows, i.e. exact products accumulated in fp32, as an fp32 GEMM
//       would, at bf16 matrix-core rate.
//       fp32: v_mfma_f32_16x16x4f32 on the fp32 products.
//     Partial sums are always added in a fixed order (wave order in LDS, then
//     slice order), so results do not depend on scheduling.  The top-k and
//     skip decisions never see bf16-rounded activations.
//     A CU keeps only a few tens of KB of loads in flight, so one workgroup
//     reading all of W_r is latency-bound.  Large batches (> 16 chunks) run one
//     fused workgroup of 8 waves per chunk (every CU busy anyway; above 256
//     chunks in bf16, one per chunk pair, route_pair_kernel); small
//     batches first spread W_r over (chunk, K slice) workgroups that write
//     partial logits, and the per-chunk kernel adds the slices.
//  2. Selection (waves 0-3, one token per 16-lane group, lane i holds slot i):
//     top-k by k rounds of a 16-lane arg-max on DPP row rotations (ties go to
//     the lower expert id; a batch of one token instead ranks every expert's
//     key against the others with all 512 threads), gates g = exp(z_i - z_1) / sum_j exp(z_j - z_1)
//     over the k selected logits (the softmax over all N experts cancels in
//     the renormalised gate), then Alg. 4 with 16-lane sums.  For the dispatch
//     plan each kept slot gets its rank among this chunk's kept slots of the
//     same expert in token order (from a 16-bit token mask per expert in LDS)
//     and the chunk's per-expert counts are written; no global atomics.
//     Meanwhile waves 4-7 write x_in = x * rstd * gamma in the GEMM dtype.
#include "ace_internal.h"

namespace ace {

namespace {

constexpr int kTok = kRouteTokens;  // tokens per router workgroup / plan chunk

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
    *reinterpret_cast<uint4 *>(p) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                               pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
  }
};


constexpr int kWaves = 8;

// value of the lane n places further round this lane's 16-lane row (DPP row_ror;
// a rotation never leaves the row, so bound_ctrl never applies and no "old"
// value has to be set up)
template <int n> __device__ __forceinline__ int row_ror(int v) {
  return __builtin_amdgcn_mov_dpp(v, 0x120 + n, 0xF, 0xF, true);
}
template <int n> __device__ __forceinline__ float row_ror(float v) {
  return __int_as_float(row_ror<n>(__float_as_int(v)));
}

// sum over the 16-lane row; a + b == b + a, so every lane ends with the same bits
__device__ __forceinline__ float group_sum(float v) {
  v += row_ror<8>(v);
  v += row_ror<4>(v);
  v += row_ror<2>(v);
  v += row_ror<1>(v);
  return v;
}

// Top-k keys: (logit, expert) as one 64-bit integer whose order is the
// selection order (larger logit first, then lower expert id); 0 = no candidate.
__device__ __forceinline__ uint64_t topk_key(float z, int e) {
  uint32_t u = __float_as_uint(z + 0.0f);  // -0 -> +0, so equal logits tie on the expert id
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | static_cast<uint32_t>(~e);
}
__device__ __forceinline__ float key_logit(uint64_t key) {
  const uint32_t u = static_cast<uint32_t>(key >> 32);
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}
__device__ __forceinline__ int key_expert(uint64_t key) { return static_cast<int>(~static_cast<uint32_t>(key)); }

// maximum over the 16-lane row, in every lane: the maximum high word, then the
// maximum low word among the lanes holding it (the same key as a 64-bit
// maximum; a valid key's low word ~expert is never 0)
__device__ __forceinline__ uint64_t row_max64(uint64_t v) {
  const uint32_t hi = static_cast<uint32_t>(v >> 32), lo = static_cast<uint32_t>(v);
  uint32_t m = hi;
  m = max(m, static_cast<uint32_t>(row_ror<8>(static_cast<int>(m))));
  m = max(m, static_cast<uint32_t>(row_ror<4>(static_cast<int>(m))));
  m = max(m, static_cast<uint32_t>(row_ror<2>(static_cast<int>(m))));
  m = max(m, static_cast<uint32_t>(row_ror<1>(static_cast<int>(m))));
  uint32_t l = hi == m ? lo : 0u;
  l = max(l, static_cast<uint32_t>(row_ror<8>(static_cast<int>(l))));
  l = max(l, static_cast<uint32_t>(row_ror<4>(static_cast<int>(l))));
  l = max(l, static_cast<uint32_t>(row_ror<2>(static_cast<int>(l))));
  l = max(l, static_cast<uint32_t>(row_ror<1>(static_cast<int>(l))));
  return (static_cast<uint64_t>(m) << 32) | l;
}

// bitonic sort, descending, of n (a power of two) keys in registers
template <int n> __device__ __forceinline__ void sort_desc(uint64_t (&a)[n]) {
#pragma unroll
  for (int blk = 2; blk <= n; blk <<= 1)
#pragma unroll
    for (int j = blk >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < n; ++i) {
        const int l = i ^ j;
        if (l > i) {
          const uint64_t x = a[i], y = a[l];
          const bool sw = ((i & blk) == 0) ? (x < y) : (x > y);
          a[i] = sw ? y : x;
          a[l] = sw ? x : y;
        }
      }
}

// number of lanes of this 16-lane group with b set
__device__ __forceinline__ int group_count(bool b) {
  const unsigned long long m = __ballot(b);
  return __popcll((m >> (threadIdx.x & 48)) & 0xFFFFull);
}

// One 32-wide K block of a lane: its 8 consecutive k of the token row, of gamma
// and of the router row of each of its NT experts (expert 16 f + lane % 16).
// Lane group g = lane / 16 supplies k = 32 j + 8 g + i (i = 0..7) to both MFMA
// operands: the A/B fragment layout of v_mfma_f32_16x16x32_bf16, and for
// v_mfma_f32_16x16x4f32 instruction i takes element i of every lane.
template <typename T, int NT> struct Stage {
  typename Oct<T>::raw x, g, w[NT];
};

template <typename T, int NT>
__device__ __forceinline__ void load_stage(Stage<T, NT> &st, const T *xrow, const T *gl, const T *wl,
                                           const int (&woff)[NT], int k) {
  st.x = Oct<T>::load(xrow + k);
  st.g = Oct<T>::load(gl + k);
#pragma unroll
  for (int f = 0; f < NT; ++f) st.w[f] = Oct<T>::load(wl + woff[f] + k);
}

// live = false: the stage holds a clamped (already counted) block; its
// activations are taken as zero so the MFMAs need no branch
// bf16 fragments arrive row-major: lane l holds 16 bytes (l % 4) of the 64 of
// row l / 4, so four consecutive lanes read one contiguous 64-byte run (MFMA
// operand order, lane l -> row l % 16, spreads every 16 lanes over 16 rows and
// streams about 3x slower from L2).  ds_bpermute moves them to operand order:
// lane l takes the data of lane 4 (l % 16) + l / 16.
__device__ __forceinline__ uint4 to_operand_order(const uint4 v) {
  const int lane = threadIdx.x & 63;
  const int src = (4 * (lane & 15) + (lane >> 4)) << 2;
  return make_uint4(static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src, static_cast<int>(v.x))),
                    static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src, static_cast<int>(v.y))),
                    static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src, static_cast<int>(v.z))),
                    static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(src, static_cast<int>(v.w))));
}

template <int NT>
__device__ __forceinline__ void mma_stage(const Stage<bf16_t, NT> &st, f32x4_t (&acc)[NT], float &ss, bool live) {
  float xv[8], gv[8];
  const uint4 xr = live ? to_operand_order(st.x) : make_uint4(0u, 0u, 0u, 0u);
  Oct<bf16_t>::cvt(xr, xv);
  Oct<bf16_t>::cvt(st.g, gv);
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t h[2], l[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const float xe = xv[2 * q + u];
      ss = fmaf(xe, xe, ss);
      const float p = xe * gv[2 * q + u];  // exact: two 8-bit significands
      const uint32_t pb = __float_as_uint(p) & 0xFFFF0000u;
      h[u] = pb;
      l[u] = __float_as_uint(p - __uint_as_float(pb));  // exact, <= 8 significant bits
    }
    hi[q] = (h[0] >> 16) | h[1];
    lo[q] = (l[0] >> 16) | (l[1] & 0xFFFF0000u);
  }
  const bf16x8_t ahi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
  const bf16x8_t alo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
  bf16x8_t w[NT];
#pragma unroll
  for (int f = 0; f < NT; ++f) w[f] = __builtin_bit_cast(bf16x8_t, to_operand_order(st.w[f]));
#pragma unroll
  for (int f = 0; f < NT; ++f) acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, w[f], acc[f], 0, 0, 0);
#pragma unroll
  for (int f = 0; f < NT; ++f) acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, w[f], acc[f], 0, 0, 0);
}

template <int NT>
__device__ __forceinline__ void mma_stage(const Stage<float, NT> &st, f32x4_t (&acc)[NT], float &ss, bool live) {
  float xv[8], gv[8], p[8];
  Oct<float>::cvt(st.x, xv);
#pragma unroll
  for (int i = 0; i < 8; ++i) xv[i] = live ? xv[i] : 0.f;
  Oct<float>::cvt(st.g, gv);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    ss = fmaf(xv[i], xv[i], ss);
    p[i] = xv[i] * gv[i];
  }
#pragma unroll
  for (int f = 0; f < NT; ++f) {
    float wv[8];
    Oct<float>::cvt(st.w[f], wv);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(p[i], wv[i], acc[f], 0, 0, 0);
  }
}

// K blocks loaded together per wave: as many as fit in about 160 VGPRs, at most 4
template <typename T, int NT> struct Depth {
  static constexpr int regs = (2 + NT) * static_cast<int>(sizeof(typename Oct<T>::raw)) / 4;
  static constexpr int fit = 160 / regs;
  static constexpr int value = fit >= 4 ? 4 : fit >= 1 ? fit : 1;
  // register stages of the pipelined loop: what is left of 256 VGPRs after the
  // accumulators (4 NT) and one stage's operands in flight to the MFMAs (4 NT + 48)
  static constexpr int ring_fit = (256 - 8 * NT - 48) / regs;
  static constexpr int ring = ring_fit >= 4 ? 4 : ring_fit;
};

// Blocks jfirst + step i (i < cnt, cnt = blocks below jend) of one wave, in
// the order i = rot, rot + 1, ... (mod cnt): workgroups that start together
// use different rotations so they do not all request the same router rows at
// once.  Sums run over the blocks in that fixed order.  When at least two
// stages fit in registers, the blocks stream through a ring of D stages: block
// i + D - 1 is requested before block i is multiplied, so D - 1 blocks' loads
// stay in flight behind the MFMAs (the compiler's vmcnt waits follow the issue
// order).  Otherwise each round loads D blocks, then multiplies them; rounds
// past the end load the last block again and zero its activations in the
// multiply, so every load is unconditional.
template <typename T, int NT>
__device__ __forceinline__ void accumulate_logits(const T *xrow, const T *gl, const T *wl, const int (&woff)[NT],
                                                  int jfirst, int jend, int step, int rot, f32x4_t (&acc)[NT],
                                                  float &ss) {
  const int cnt = jend > jfirst ? (jend - jfirst + step - 1) / step : 0;
  if (cnt == 0) return;
  rot %= cnt;
  auto kof = [&](int i) {
    int b = i + rot;
    b = b >= cnt ? b - cnt : b;
    return 32 * (jfirst + b * step);
  };
  if constexpr (Depth<T, NT>::ring >= 2) {
    constexpr int D = Depth<T, NT>::ring;
    Stage<T, NT> st[D];
#pragma unroll
    for (int u = 0; u < D - 1; ++u)
      if (u < cnt) load_stage<T, NT>(st[u], xrow, gl, wl, woff, kof(u));
    for (int i0 = 0; i0 < cnt; i0 += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        const int i = i0 + u;
        if (i >= cnt) break;
        if (i + D - 1 < cnt) load_stage<T, NT>(st[(u + D - 1) % D], xrow, gl, wl, woff, kof(i + D - 1));
        mma_stage<NT>(st[u], acc, ss, true);
      }
    }
  } else {
    constexpr int D = Depth<T, NT>::value;
    for (int i0 = 0; i0 < cnt; i0 += D) {
      Stage<T, NT> st[D];
#pragma unroll
      for (int u = 0; u < D; ++u) load_stage<T, NT>(st[u], xrow, gl, wl, woff, kof(min(i0 + u, cnt - 1)));
#pragma unroll
      for (int u = 0; u < D; ++u) mma_stage<NT>(st[u], acc, ss, i0 + u < cnt);
    }
  }
}

// One wave's partial logits of blocks jfirst, jfirst + step, ... < jend for
// the 16 tokens from t0, into zred[token][expert] and ssred[token] (LDS).
template <typename T, int NT, int ZS, bool ONE_BLOCK_PATH>
__device__ __forceinline__ void wave_logits(const RouteArgs &a, int t0, int jfirst, int jend, int step, int rot,
                                            float (*zred)[ZS], float *ssred) {
  const T *x = static_cast<const T *>(a.x);
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int d = a.d, N = a.N;
  // row and 8-element chunk this lane loads: bf16 rows are loaded row-major
  // (row lane / 4, chunk lane % 4) and permuted into operand order in
  // mma_stage; fp32 rows are loaded in operand order (row lane % 16, chunk lane / 16)
  constexpr bool kRowMajor = sizeof(T) == 2;
  const int lrow = kRowMajor ? lane >> 2 : r16, lchunk = kRowMajor ? lane & 3 : grp;
  const int trow = min(t0 + lrow, a.T - 1);  // rows past the batch repeat the last token
  const T *xrow = x + static_cast<size_t>(trow) * d + lchunk * 8;
  const T *gl = static_cast<const T *>(a.gamma) + grp * 8;
  const T *wl = static_cast<const T *>(a.w_router) + lchunk * 8;
  int woff[NT];
#pragma unroll
  for (int f = 0; f < NT; ++f) woff[f] = min(16 * f + lrow, N - 1) * d;
  f32x4_t acc[NT];
#pragma unroll
  for (int f = 0; f < NT; ++f) acc[f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float ss = 0.f;
  if (ONE_BLOCK_PATH && jfirst < jend && jfirst + step >= jend) {
    // exactly one block (decode-sized K slices): one load round, no repeats
    Stage<T, NT> st;
    load_stage<T, NT>(st, xrow, gl, wl, woff, 32 * jfirst);
    mma_stage<NT>(st, acc, ss, true);
  } else {
    accumulate_logits<T, NT>(xrow, gl, wl, woff, jfirst, jend, step, rot, acc, ss);
  }
  // D[row = token 4 grp + i][col = expert 16 f + r16]
#pragma unroll
  for (int f = 0; f < NT; ++f)
#pragma unroll
    for (int i = 0; i < 4; ++i) zred[grp * 4 + i][16 * f + r16] = acc[f][i];
  // lanes of token r16 are r16 + 16 g
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  if (grp == 0) ssred[r16] = ss;
}

constexpr int kPartWaves = 4;

// Small batches: grid (chunks, K slices); workgroup (c, s) writes the partial
// logits zpart[s][t][0..zstride) (before the RMS scale) and the partial sums
// of squares sspart[s][t] of slice s for the tokens of chunk c.
template <typename T, int NT>
__global__ __launch_bounds__(256) void route_partial_kernel(RouteArgs a) {
  constexpr int NP = NT * 16;
  __shared__ float zred[kPartWaves][kTok][NP + 1];
  __shared__ float ssred[kPartWaves][kTok];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int t0 = blockIdx.x * kTok;
  const int s = blockIdx.y;
  const int nbs = (a.d >> 5) / a.ksplit;  // blocks per slice
  wave_logits<T, NT, NP + 1, true>(a, t0, s * nbs + wave, (s + 1) * nbs, kPartWaves, blockIdx.x, zred[wave],
                                   ssred[wave]);
  __syncthreads();
  const size_t plane = static_cast<size_t>(s) * a.T;
  for (int idx = tid; idx < kTok * NP; idx += 256) {
    const int tl = idx / NP;
    const int e = idx - tl * NP;
    if (t0 + tl >= a.T) continue;
    float z = 0.f;
#pragma unroll
    for (int w = 0; w < kPartWaves; ++w) z += zred[w][tl][e];
    a.zpart[(plane + t0 + tl) * a.zstride + e] = z;
  }
  if (tid < kTok && t0 + tid < a.T) {
    float ss = 0.f;
#pragma unroll
    for (int w = 0; w < kPartWaves; ++w) ss += ssred[w][tid];
    a.sspart[plane + t0 + tid] = ss;
  }
}

// One chunk (at most 16 tokens): its only select workgroup writes the plan
// straight from the per-expert token masks in LDS and each kept slot's rank
// (held by the slot's own lane), with no global re-read: row = offsets[e] +
// rank, the rows the plan kernels give.  Several chunks: the plan kernels of
// dispatch.hip follow.
__device__ __forceinline__ void plan_one_chunk(const RouteArgs &a, const uint32_t *emask, bool kept, int e_mine,
                                               int t, int sub, int rank) {
  __shared__ int off1[kMaxN + 1];
  const int tid = threadIdx.x, lane = tid & 63;
  const int N = a.N;
  if (tid < 64) {
    // exclusive scans of the counts and tile counts (N <= 256: four per lane)
    int s = 0, st = 0, loc[4], loct[4], c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane * 4 + j;
      c[j] = e < N ? __popc(emask[e]) : 0;
      loc[j] = s;
      loct[j] = st;
      s += c[j];
      st += (c[j] + kTileM - 1) / kTileM;
    }
    int inc = s, inct = st;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(inc, o), vt = __shfl_up(inct, o);
      if (lane >= o) {
        inc += v;
        inct += vt;
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane * 4 + j;
      if (e < N) {
        const int off = inc - s + loc[j], toff = inct - st + loct[j];
        off1[e] = off;
        a.counts[e] = c[j];
        a.offsets[e] = off;
        for (int q = 0; q * kTileM < c[j]; ++q) {
          a.tile_expert[toff + q] = e;
          a.tile_row0[toff + q] = off + q * kTileM;
          a.tile_rows[toff + q] = min(kTileM, c[j] - q * kTileM);
        }
      }
    }
    if (lane == 63) {
      a.offsets[N] = inc;
      a.n_tiles[0] = inct;
    }
  }
  __syncthreads();
  if (kept) {
    const int row = off1[e_mine] + rank;
    a.perm[row] = t;
    a.slot_row[static_cast<size_t>(t) * a.k + sub] = row;
  }
}

// NT = number of 16-expert tiles covered (N <= 16 * NT).  SPLIT: the logits
// come from route_partial_kernel's K slices; otherwise the 8 waves compute
// them here over all of K.
// Top-k, gates and Alg. 4 for token t (valid if tvalid) held by one 16-lane
// group, lane `sub` holding slot `sub` (sub < k); zrow = the token's N logits
// in LDS.  Writes the token's routing outputs; returns the expert and keep
// decision of this lane's slot through my_e / my_kept.
// top (or nullptr): the token's k keys in selection order, already chosen.
template <int NT>
__device__ __forceinline__ void select_token(const RouteArgs &a, const float *zrow, int t, bool tvalid, int sub,
                                             const float *a_gsp_s, const float *a_rcr_s, int &my_e, bool &my_kept,
                                             const uint64_t *top = nullptr) {
  const int N = a.N;
  const int k = a.k;
  uint64_t mykey = 0, topkey = 0;
  if (top) {
    topkey = top[0];
    if (sub < k) mykey = top[sub];
  } else {
  // this lane's candidates, experts sub + 16 q, sorted; it can lose at most k <= 8 of them
  uint64_t cand[NT];
#pragma unroll
  for (int q = 0; q < NT; ++q) {
    const int e = sub + 16 * q;
    cand[q] = (e < N) ? topk_key(zrow[e], e) : 0ull;
  }
  sort_desc<NT>(cand);
  constexpr int L = NT < kMaxK ? NT : kMaxK;
  uint64_t head[L];
#pragma unroll
  for (int q = 0; q < L; ++q) head[q] = cand[q];
  // k rounds: the row maximum of the lanes' heads is the next slot; the lane
  // that held it pops its head
#pragma unroll
  for (int i = 0; i < kMaxK; ++i) {
    if (i >= k) break;
    const uint64_t m = row_max64(head[0]);
    if (i == 0) topkey = m;
    if (sub == i) mykey = m;
    const bool win = head[0] == m;
#pragma unroll
    for (int q = 0; q + 1 < L; ++q) head[q] = win ? head[q + 1] : head[q];
    head[L - 1] = win ? 0ull : head[L - 1];
  }
  }
  const bool slot = sub < k;
  const int se = slot ? key_expert(mykey) : 0;  // this lane's slot: expert and logit
  const float sz = key_logit(mykey), ztop = key_logit(topkey);
  // renormalised top-k gate
  const float ge = slot ? expf(sz - ztop) : 0.f;
  const float g = ge / group_sum(ge);
  // Alg. 4: s = g * A(e); p = s / (sum s + eps); ACE: c = max(p_GSP, p_RCR)
  const float sg = slot ? g * a_gsp_s[se] : 0.f;
  const float sr = slot ? g * a_rcr_s[se] : 0.f;
  const float pg = sg / (group_sum(sg) + a.eps);
  const float pr = sr / (group_sum(sr) + a.eps);
  float c;
  switch (a.fusion) {
    case 1: c = fminf(pg, pr); break;           // either view low (union)
    case 2: c = (pg + pr) * 0.5f; break;        // mean of the views
    case 3: c = pg; break;                      // GSP only
    case 4: c = pr; break;                      // RCR only
    case 5: {                                   // router score: the p of a table of ones
      const float gs = slot ? g : 0.f;
      c = gs / (group_sum(gs) + a.eps);
      break;
    }
    default: c = fmaxf(pg, pr);                 // ACE: both views low (intersection)
  }
  // slot 0 is the top-1 expert, never skipped
  const bool skip = !a.skip_disable && sub > 0 && c < a.tau;
  bool kept = slot && !skip;
  const int nkept = group_count(kept);
  if (!a.skip_disable && nkept < a.m_min) {
    // restore skipped slots by descending c (ties -> lower slot) up to m_min
    int rank = 0;
#pragma unroll 1
    for (int jj = 0; jj < k; ++jj) {
      const float cj = __shfl(c, jj, 16);
      const int kj = __shfl(kept ? 1 : 0, jj, 16);
      if (!kj && jj != sub && (cj > c || (cj == c && jj < sub))) ++rank;
    }
    kept = kept || (slot && rank < a.m_min - nkept);
  }
  const float zgate = group_sum(kept ? g : 0.f) + a.eps;
  if (tvalid && slot) {
    const size_t o = static_cast<size_t>(t) * k + sub;
    a.topk_idx[o] = se;
    a.keep[o] = kept ? 1 : 0;
    a.gates[o] = a.skip_disable ? g : (kept ? g / zgate : 0.f);
    if (a.scores) a.scores[o] = c;
    if (!kept) a.slot_row[o] = -1;
    my_e = se;
    my_kept = kept;
  }
}

// One-token top-k by rank (route_kernel): NC slices of JL experts each, NC * NP
// <= 512 threads, one (expert, slice) pair per thread.
template <int NP> struct RankSlices {
  static constexpr int JL = NP * NP / 512 > 1 ? NP * NP / 512 : 1;
  static constexpr int NC = NP / JL;
  static_assert(NC * JL == NP && NC * NP <= 512, "slices cover the experts");
};

// ONE (with SPLIT): a batch of one token, its top-k by rank.
template <typename T, int NT, bool SPLIT, bool ONE = false>
__global__ __launch_bounds__(512) void route_kernel(RouteArgs a) {
  constexpr int NP = NT * 16;
  const T *__restrict__ x = static_cast<const T *>(a.x);
  const T *__restrict__ gamma = static_cast<const T *>(a.gamma);
  T *__restrict__ xn = static_cast<T *>(a.xn);

  __shared__ float zred[SPLIT ? 1 : kWaves][kTok][NP + 1];  // per-wave partial logits; slot 0 ends as z
  __shared__ float ssred[kWaves][kTok];
  __shared__ float rstd_s[kTok];
  __shared__ uint32_t emask[NP];
  __shared__ float a_gsp_s[NP], a_rcr_s[NP];
  __shared__ uint64_t key_s[ONE ? NP : 1], top_s[ONE ? kMaxK : 1];  // one-token top-k by rank
  __shared__ uint16_t rank_s[ONE ? RankSlices<NP>::NC : 1][ONE ? NP : 1];
  static_assert(512 % NP == 0, "a thread meets one expert column in the logits reduction");

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar loop control
  const int t0 = blockIdx.x * kTok;
  const int d = a.d, N = a.N, nt = a.T;
  if (tid < NP) {
    emask[tid] = 0u;
    a_gsp_s[tid] = tid < N ? a.a_gsp[tid] : 0.f;
    a_rcr_s[tid] = tid < N ? a.a_rcr[tid] : 0.f;
  }
  // router bias of this thread's expert column in the logits reduction below
  const float bias = (a.b_router && (tid % NP) < N) ? a.b_router[tid % NP] : 0.f;

  if constexpr (SPLIT) {
    // ---- 1. add the K slices' partial logits and sums of squares in slice
    // order; every load of the workgroup is issued before the first add
    constexpr int PER = (kTok * NP + 2047) / 2048;  // groups of 4 logits per thread (16-byte loads)
    float ssp[kRouteMaxSlices];
#pragma unroll
    for (int sl = 0; sl < kRouteMaxSlices; ++sl)
      ssp[sl] = (tid < kTok && sl < a.ksplit) ? a.sspart[static_cast<size_t>(sl) * nt + min(t0 + tid, nt - 1)] : 0.f;
    float4 part[PER][kRouteMaxSlices];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int idx = min(4 * tid + 2048 * u, kTok * NP - 4);
      const int tl = idx / NP;
      const int e = idx - tl * NP;
      const size_t col = static_cast<size_t>(min(t0 + tl, nt - 1)) * a.zstride + e;
#pragma unroll
      for (int sl = 0; sl < kRouteMaxSlices; ++sl)
        part[u][sl] = sl < a.ksplit ? *reinterpret_cast<const float4 *>(a.zpart + static_cast<size_t>(sl) * nt * a.zstride + col)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (tid < kTok) {
      float ssum = 0.f;
#pragma unroll
      for (int sl = 0; sl < kRouteMaxSlices; ++sl) ssum += ssp[sl];
      rstd_s[tid] = 1.0f / sqrtf(ssum / static_cast<float>(d) + a.rms_eps);
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int idx = 4 * tid + 2048 * u;
      if (idx < kTok * NP) {
        const int tl = idx / NP;
        float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int sl = 0; sl < kRouteMaxSlices; ++sl) {
          z.x += part[u][sl].x;
          z.y += part[u][sl].y;
          z.z += part[u][sl].z;
          z.w += part[u][sl].w;
        }
        float *zr = &zred[0][tl][idx - tl * NP];
        zr[0] = z.x;
        zr[1] = z.y;
        zr[2] = z.z;
        zr[3] = z.w;
      }
    }
    __syncthreads();
    for (int idx = tid; idx < kTok * NP; idx += 512) {
      const int tl = idx / NP;
      const int e = idx - tl * NP;
      zred[0][tl][e] = zred[0][tl][e] * rstd_s[tl] + bias;
    }
    __syncthreads();
    if constexpr (ONE) {
      // one token (batch 1): its top-k by rank.  Expert i's rank is the number of
      // keys above its key (keys are distinct, so the ranks are a permutation and
      // ranks 0..k-1 are the top-k in selection order); the 512 threads each
      // count over a slice of the experts, a few dozen independent comparisons
      // instead of the 16-lane sort and arg-max rounds' dependent chain
      constexpr int JL = RankSlices<NP>::JL, NC = RankSlices<NP>::NC;  // experts per slice, slices
      if (tid < NP) key_s[tid] = tid < N ? topk_key(zred[0][0][tid], tid) : 0ull;
      __syncthreads();
      const int i = tid % NP, c = tid / NP;
      const uint64_t ki = key_s[i];
      if (c < NC) {
        int r = 0;
#pragma unroll 8
        for (int jj = 0; jj < JL; ++jj) r += key_s[c * JL + jj] > ki ? 1 : 0;
        rank_s[c][i] = static_cast<uint16_t>(r);
      }
      __syncthreads();
      if (tid < N) {
        int rr = 0;
#pragma unroll
        for (int q = 0; q < NC; ++q) rr += rank_s[q][tid];
        if (rr < a.k) top_s[rr] = ki;
      }
      __syncthreads();
    }
  } else {
    // ---- 1. logits over all K: wave w takes blocks w, w + 8, ...
    // workgroups are dealt to the 8 XCDs round-robin: rotate by the index on the XCD
    wave_logits<T, NT, NP + 1, false>(a, t0, wave, d >> 5, kWaves, blockIdx.x >> 3, zred[wave], ssred[wave]);
    __syncthreads();
    if (tid < kTok) {
      float ssum = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) ssum += ssred[w][tid];
      rstd_s[tid] = 1.0f / sqrtf(ssum / static_cast<float>(d) + a.rms_eps);
    }
    __syncthreads();
    for (int idx = tid; idx < kTok * NP; idx += 512) {
      const int tl = idx / NP;
      const int e = idx - tl * NP;
      float z = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) z += zred[w][tl][e];
      zred[0][tl][e] = z * rstd_s[tl] + bias;
    }
    __syncthreads();
  }

  int my_e = -1;  // expert of this lane's slot (lane sub < k), -1 if none
  bool my_kept = false;
  const int sub = lane & 15;
  const int tl = wave * 4 + (lane >> 4);
  const int t = t0 + tl;
  if (wave >= 4) {
    // ---- x_in = x * rstd * gamma for the expert GEMMs (waves 4-7)
    const int d8 = d >> 3;
    for (int c8 = tid - 256; c8 < d8; c8 += 256) {
      // all 16 rows in flight at once (rows past the batch load the last token, unused)
      typename Oct<T>::raw xr[kTok];
#pragma unroll
      for (int u = 0; u < kTok; ++u) xr[u] = Oct<T>::load(x + static_cast<size_t>(min(t0 + u, nt - 1)) * d + 8 * c8);
      float gv[8];
      Oct<T>::cvt(Oct<T>::load(gamma + 8 * c8), gv);
#pragma unroll
      for (int u = 0; u < kTok; ++u) {
        if (t0 + u >= nt) break;
        float xv[8], av[8];
        Oct<T>::cvt(xr[u], xv);
        const float rs = rstd_s[u];
#pragma unroll
        for (int i = 0; i < 8; ++i) av[i] = (xv[i] * rs) * gv[i];
        Oct<T>::store(xn + static_cast<size_t>(t0 + u) * d + 8 * c8, av);
      }
    }
  } else {
    // ---- 2. top-k, gates and Alg. 4 (waves 0-3): one token per 16-lane
    // group, lane `sub` holds slot `sub` (sub < k)
    select_token<NT>(a, zred[0][tl], t, t < nt, sub, a_gsp_s, a_rcr_s, my_e, my_kept,
                     ONE ? top_s : nullptr);
  }
  // ---- per-expert token masks of this chunk -> local ranks and counts
  if (my_kept) atomicOr(&emask[my_e], 1u << tl);
  __syncthreads();
  const int my_rank = my_kept ? __popc(emask[my_e] & ((1u << tl) - 1u)) : 0;
  if constexpr (SPLIT) {
    if (gridDim.x == 1) {
      plan_one_chunk(a, emask, my_kept, my_e, t, sub, my_rank);
      return;
    }
  }
  if (my_kept) a.local_rank[static_cast<size_t>(t) * a.k + sub] = static_cast<uint8_t>(my_rank);
  for (int e = tid; e < N; e += 512)
    a.chunk_count[static_cast<size_t>(blockIdx.x) * N + e] = static_cast<uint8_t>(__popc(emask[e]));
}

// Batches of more than 256 chunks (bf16): one workgroup of 8 waves per pair of
// chunks (32 tokens).  Each router-row fragment a wave loads feeds the MFMAs of
// both 16-token tiles, so every CU streams W_r once per two chunks, and the
// grid is one round of workgroups instead of two.  The waves split the experts
// in two halves (NT >= 2) and K in four groups: wave w multiplies expert tiles
// (w % 2) NT/2 .. and K blocks w/2, w/2 + 4, ..., so its accumulators and a
// register stage stay small enough for a ring of stages (block i + D - 1 is
// requested before block i is multiplied).  Fixed summation: blocks in order
// within a wave, then the four K groups in order; then selection (waves 0-3:
// the first chunk's tokens, waves 4-7: the second's), x_in for the 32 rows, and
// per-chunk ranks and counts.
constexpr int kPairWaves = 8;
template <int NTW> struct PairStage {
  uint4 x[2], g, w[NTW];
};
// register stages per wave within 2 waves per SIMD: accumulators 8 NTW, the
// operands of one stage on their way to the MFMAs 4 (NTW + 2), about 40 more
template <int NTW> struct PairDepth {
  static constexpr int fit = (256 - 8 * NTW - 4 * (NTW + 2) - 40) / ((3 + NTW) * 4);
  static constexpr int value = fit >= 4 ? 4 : fit >= 1 ? fit : 1;
};

template <int NT>
__global__ __launch_bounds__(512) void route_pair_kernel(RouteArgs a) {
  constexpr int NP = NT * 16, TOK = 2 * kTok;
  constexpr int EH = NT >= 2 ? 2 : 1;       // expert groups
  constexpr int NTW = NT / EH;              // expert tiles per wave
  constexpr int KG = kPairWaves / EH;       // K groups
  constexpr int D = PairDepth<NTW>::value;
  static_assert(512 % NP == 0, "a thread meets one expert column in the logits reduction");
  __shared__ float zred[KG][TOK][NP + 1];   // K group kg's partial logits (all experts)
  __shared__ float ssred[KG][TOK];
  __shared__ float rstd_s[TOK];
  __shared__ uint32_t emask[2][NP];
  __shared__ float a_gsp_s[NP], a_rcr_s[NP];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, grp = lane >> 4;
  const int t0 = blockIdx.x * TOK;
  const int d = a.d, N = a.N, nt = a.T;
  const int G = (nt + kTok - 1) / kTok;
  const bf16_t *x = static_cast<const bf16_t *>(a.x);
  const bf16_t *gamma = static_cast<const bf16_t *>(a.gamma);
  bf16_t *xn = static_cast<bf16_t *>(a.xn);
  if (tid < NP) {
    emask[0][tid] = emask[1][tid] = 0u;
    a_gsp_s[tid] = tid < N ? a.a_gsp[tid] : 0.f;
    a_rcr_s[tid] = tid < N ? a.a_rcr[tid] : 0.f;
  }
  const float bias = (a.b_router && (tid % NP) < N) ? a.b_router[tid % NP] : 0.f;

  // ---- 1. logits of both token tiles
  {
    const int eh = wave % EH, kg = wave / EH;
    const int lrow = lane >> 2, lchunk = lane & 3;  // row-major fragment loads
    const bf16_t *xrow[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) xrow[c] = x + static_cast<size_t>(min(t0 + 16 * c + lrow, nt - 1)) * d + lchunk * 8;
    const bf16_t *gl = gamma + grp * 8;
    const bf16_t *wl = static_cast<const bf16_t *>(a.w_router) + lchunk * 8;
    int woff[NTW];
#pragma unroll
    for (int f = 0; f < NTW; ++f) woff[f] = min(16 * (eh * NTW + f) + lrow, N - 1) * d;
    f32x4_t acc[2][NTW];
    float ss[2] = {0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int f = 0; f < NTW; ++f) acc[c][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int nb = d >> 5;
    const int cnt = nb > kg ? (nb - kg + KG - 1) / KG : 0;
    const int rot = cnt > 0 ? static_cast<int>((blockIdx.x >> 3) % cnt) : 0;
    auto load = [&](PairStage<NTW> &st, int i) {
      int b = i + rot;
      b = b >= cnt ? b - cnt : b;
      const int k = 32 * (kg + b * KG);
#pragma unroll
      for (int c = 0; c < 2; ++c) st.x[c] = *reinterpret_cast<const uint4 *>(xrow[c] + k);
      st.g = *reinterpret_cast<const uint4 *>(gl + k);
#pragma unroll
      for (int f = 0; f < NTW; ++f) st.w[f] = *reinterpret_cast<const uint4 *>(wl + woff[f] + k);
    };
    auto mma = [&](const PairStage<NTW> &st) {
      float gv[8];
      Oct<bf16_t>::cvt(st.g, gv);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        float xv[8];
        Oct<bf16_t>::cvt(to_operand_order(st.x[c]), xv);
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t h[2], l[2];
#pragma unroll
          for (int v = 0; v < 2; ++v) {
            const float xe = xv[2 * q + v];
            ss[c] = fmaf(xe, xe, ss[c]);
            const float pr = xe * gv[2 * q + v];  // exact: two 8-bit significands
            const uint32_t pb = __float_as_uint(pr) & 0xFFFF0000u;
            h[v] = pb;
            l[v] = __float_as_uint(pr - __uint_as_float(pb));  // exact, <= 8 significant bits
          }
          hi[q] = (h[0] >> 16) | h[1];
          lo[q] = (l[0] >> 16) | (l[1] & 0xFFFF0000u);
        }
        const bf16x8_t ahi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
        const bf16x8_t alo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
#pragma unroll
        for (int f = 0; f < NTW; ++f) {
          const bf16x8_t w = __builtin_bit_cast(bf16x8_t, to_operand_order(st.w[f]));
          acc[c][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, w, acc[c][f], 0, 0, 0);
          acc[c][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, w, acc[c][f], 0, 0, 0);
        }
      }
    };
    PairStage<NTW> st[D];
#pragma unroll
    for (int u = 0; u < D - 1; ++u)
      if (u < cnt) load(st[u], u);
    for (int i0 = 0; i0 < cnt; i0 += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        const int i = i0 + u;
        if (i >= cnt) break;
        if (i + D - 1 < cnt) load(st[(u + D - 1) % D], i + D - 1);
        mma(st[u]);
      }
    }
    // D[row = token 4 grp + i][col = expert 16 f + r16] of each token tile into
    // the K group's slot; the sums of squares once per K group (expert group 0)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      float v = ss[c];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (eh == 0 && grp == 0) ssred[kg][16 * c + r16] = v;
    }
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int f = 0; f < NTW; ++f)
#pragma unroll
        for (int i = 0; i < 4; ++i) zred[kg][16 * c + grp * 4 + i][16 * (eh * NTW + f) + r16] = acc[c][f][i];
  }
  __syncthreads();
  if (tid < TOK) {
    float ssum = 0.f;
#pragma unroll
    for (int w = 0; w < KG; ++w) ssum += ssred[w][tid];
    rstd_s[tid] = 1.0f / sqrtf(ssum / static_cast<float>(d) + a.rms_eps);
  }
  __syncthreads();
  for (int idx = tid; idx < TOK * NP; idx += 512) {
    const int tl = idx / NP;
    const int e = idx - tl * NP;
    float z = 0.f;
#pragma unroll
    for (int w = 0; w < KG; ++w) z += zred[w][tl][e];
    zred[0][tl][e] = z * rstd_s[tl] + bias;
  }
  __syncthreads();

  // ---- 2. selection: waves 0-3 the first chunk's tokens, waves 4-7 the second's,
  // one token per 16-lane group
  const int sub = lane & 15;
  const int p = wave >> 2;                        // this wave's chunk
  const int tlc = (wave & 3) * 4 + (lane >> 4);   // token within its chunk
  int my_e = -1;
  bool my_kept = false;
  {
    const int t = t0 + 16 * p + tlc;
    select_token<NT>(a, zred[0][16 * p + tlc], t, t < nt, sub, a_gsp_s, a_rcr_s, my_e, my_kept);
  }
  // ---- 3. x_in = x * rstd * gamma for the expert GEMMs, 16 rows at a time
  const int d8 = d >> 3;
  for (int c8 = tid; c8 < 2 * d8; c8 += 512) {
    // thread pairs (c8, c8 + d8) share a column octet: rows of chunk q = c8 / d8
    const int q = c8 >= d8 ? 1 : 0, o8 = c8 - q * d8;
    float gv[8];
    Oct<bf16_t>::cvt(Oct<bf16_t>::load(gamma + 8 * o8), gv);
    {
      const int r0 = t0 + 16 * q;
      typename Oct<bf16_t>::raw xr[kTok];
#pragma unroll
      for (int u = 0; u < kTok; ++u) xr[u] = Oct<bf16_t>::load(x + static_cast<size_t>(min(r0 + u, nt - 1)) * d + 8 * o8);
#pragma unroll
      for (int u = 0; u < kTok; ++u) {
        if (r0 + u >= nt) break;
        float xv[8], av[8];
        Oct<bf16_t>::cvt(xr[u], xv);
        const float rs = rstd_s[16 * q + u];
#pragma unroll
        for (int i = 0; i < 8; ++i) av[i] = (xv[i] * rs) * gv[i];
        Oct<bf16_t>::store(xn + static_cast<size_t>(r0 + u) * d + 8 * o8, av);
      }
    }
  }
  // ---- 4. per-expert token masks of each chunk -> local ranks and counts
  if (my_kept) atomicOr(&emask[p][my_e], 1u << tlc);
  __syncthreads();
  if (my_kept) {
    const int t = t0 + 16 * p + tlc;
    a.local_rank[static_cast<size_t>(t) * a.k + sub] = static_cast<uint8_t>(__popc(emask[p][my_e] & ((1u << tlc) - 1u)));
  }
  for (int i = tid; i < 2 * N; i += 512) {
    const int q = i >= N ? 1 : 0, e = i - q * N;
    const int c = 2 * blockIdx.x + q;
    if (c < G) a.chunk_count[static_cast<size_t>(c) * N + e] = static_cast<uint8_t>(__popc(emask[q][e]));
  }
}

template <typename T, int NT>
void launch_route_nt(const RouteArgs &a, hipStream_t stream) {
  const int chunks = (a.T + kTok - 1) / kTok;
  if constexpr (sizeof(T) == 2) {
    if (a.ksplit == 0 && chunks > kRoutePairMinChunks) {
      route_pair_kernel<NT><<<dim3((chunks + 1) / 2), 512, 0, stream>>>(a);
      return;
    }
  }
  if (a.ksplit > 0) {
    route_partial_kernel<T, NT><<<dim3(chunks, a.ksplit), 256, 0, stream>>>(a);
    if (a.T == 1)
      route_kernel<T, NT, true, true><<<dim3(chunks), 512, 0, stream>>>(a);
    else
      route_kernel<T, NT, true><<<dim3(chunks), 512, 0, stream>>>(a);
  } else {
    route_kernel<T, NT, false><<<dim3(chunks), 512, 0, stream>>>(a);
  }
}

template <typename T>
hipError_t launch_route_t(const RouteArgs &a, hipStream_t stream) {
  const int nt = route_expert_tiles(a.N);
  if (nt == 1)
    launch_route_nt<T, 1>(a, stream);
  else if (nt == 2)
    launch_route_nt<T, 2>(a, stream);
  else if (nt == 4)
    launch_route_nt<T, 4>(a, stream);
  else if (nt == 8)
    launch_route_nt<T, 8>(a, stream);
  else
    launch_route_nt<T, 16>(a, stream);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const RouteArgs &a, bool bf16, hipStream_t stream) {
  return bf16 ? launch_route_t<bf16_t>(a, stream) : launch_route_t<float>(a, stream);
}

}  // namespace ace
