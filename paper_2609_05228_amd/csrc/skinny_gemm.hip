// Grouped expert GEMMs for small batches (decode): at most 64 tokens, so every
// expert has at most 64 kept rows and the layer is a batch of weight-streaming
// GEMVs.  Work is split so that thousands of waves stream weights at once:
//  * a work item is one wave: one tile (expert) x 16 features (gate/up: a gate
//    block and an up block) or 32 output columns (down) x one K split;
//  * the wave loads its weight and activation MFMA fragments straight into
//    registers through a P-stage ring (no LDS, no barriers) and multiplies them
//    with v_mfma_f32_16x16x32_bf16;
//  * with one K split the epilogue writes H (SwiGLU applied) or Y in bf16;
//    with several, it writes fp32 partial sums, which swiglu_reduce_kernel (for
//    H) and the combine kernel (for Y) add in split order, so the result does
//    not depend on scheduling.
#include "ace_internal.h"

namespace ace {

namespace {

struct TileInfo {
  int e, row0, rows;
  bool valid;
};

__device__ __forceinline__ TileInfo skinny_tile(const GemmArgs &a, int grp) {
  TileInfo ti;
  if (a.dense_rows > 0) {
    ti.e = 0;
    ti.row0 = grp * kTileM;
    ti.rows = min(kTileM, a.dense_rows - ti.row0);
    ti.valid = ti.rows > 0;
  } else {
    ti.valid = grp < a.n_tiles[0];
    ti.e = ti.valid ? a.tile_expert[grp] : 0;
    ti.row0 = ti.valid ? a.tile_row0[grp] : 0;
    ti.rows = ti.valid ? a.tile_rows[grp] : 0;
  }
  return ti;
}

__device__ __forceinline__ float silu(float v) { return v / (1.0f + expf(-v)); }

// ring depth: registers for P stages of 4 weight + 2*MB activation fragments
template <int MB> struct Ring {
  static constexpr int P = MB == 1 ? 8 : MB == 2 ? 6 : 4;
};

template <int MB> struct Stage {
  uint4 b[2][2];   // [block][k half]
  uint4 a[MB][2];  // [row block][k half]
};

template <int MB>
__device__ __forceinline__ void load_stage(Stage<MB> &st, const bf16_t *const (&bsrc)[2],
                                           const bf16_t *const (&asrc)[MB], int k) {
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int h = 0; h < 2; ++h) st.b[cb][h] = *reinterpret_cast<const uint4 *>(bsrc[cb] + k + 32 * h);
#pragma unroll
  for (int mi = 0; mi < MB; ++mi)
#pragma unroll
    for (int h = 0; h < 2; ++h) st.a[mi][h] = *reinterpret_cast<const uint4 *>(asrc[mi] + k + 32 * h);
}

template <int MB>
__device__ __forceinline__ void mma_stage(const Stage<MB> &st, f32x4_t (&acc)[MB][2]) {
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
        acc[mi][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, st.a[mi][h]),
                                                              __builtin_bit_cast(bf16x8_t, st.b[cb][h]),
                                                              acc[mi][cb], 0, 0, 0);
}

template <bool GATEUP, int MB>
__device__ __forceinline__ void skinny_item(const SkinnyArgs &sa, const TileInfo &ti, int nb, int s) {
  constexpr int P = Ring<MB>::P;
  const GemmArgs &a = sa.g;
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const int K = GATEUP ? a.d : a.m;
  const int kc = K / sa.splits;
  const int kbase = s * kc;
  const int nk = kc / 64;

  const bf16_t *bsrc[2];
  if (GATEUP) {
    const size_t f = static_cast<size_t>(ti.e) * a.m + nb * 16 + r16;
    bsrc[0] = static_cast<const bf16_t *>(a.w0) + f * a.d + kbase + 8 * g;
    bsrc[1] = static_cast<const bf16_t *>(a.w1) + f * a.d + kbase + 8 * g;
  } else {
    const size_t n = static_cast<size_t>(ti.e) * a.d + nb * 32 + r16;
    bsrc[0] = static_cast<const bf16_t *>(a.w0) + n * a.m + kbase + 8 * g;
    bsrc[1] = bsrc[0] + static_cast<size_t>(16) * a.m;
  }
  const bf16_t *act = static_cast<const bf16_t *>(a.act);
  const bf16_t *asrc[MB];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
    const int row = min(mi * 16 + r16, ti.rows - 1);  // rows past the tile repeat its last row
    const int src_row = a.perm ? a.perm[ti.row0 + row] : ti.row0 + row;
    asrc[mi] = act + static_cast<size_t>(src_row) * K + kbase + 8 * g;
  }

  f32x4_t acc[MB][2];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
    acc[mi][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc[mi][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  Stage<MB> ring[P];
#pragma unroll
  for (int u = 0; u < P; ++u)
    if (u < nk) load_stage<MB>(ring[u], bsrc, asrc, u * 64);
  for (int k0 = 0; k0 < nk; k0 += P) {
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const int kt = k0 + u;
      if (kt < nk) {
        mma_stage<MB>(ring[u], acc);
        if (kt + P < nk) load_stage<MB>(ring[u], bsrc, asrc, (kt + P) * 64);
      }
    }
  }

  // epilogue: lane holds column r16 of each block, rows 4*g + q
#pragma unroll
  for (int mi = 0; mi < MB; ++mi)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int row = mi * 16 + 4 * g + q;
      if (row >= ti.rows) continue;
      const size_t r = static_cast<size_t>(ti.row0 + row);
      if (GATEUP) {
        const int f = nb * 16 + r16;
        if (sa.splits == 1) {
          static_cast<bf16_t *>(a.out)[r * a.m + f] = f32_to_bf16(silu(acc[mi][0][q]) * acc[mi][1][q]);
        } else {
          const size_t o = (static_cast<size_t>(s) * sa.rows_cap + r) * a.m + f;
          sa.part0[o] = acc[mi][0][q];
          sa.part1[o] = acc[mi][1][q];
        }
      } else {
        const int n = nb * 32 + r16;
        if (sa.splits == 1) {
          bf16_t *yr = static_cast<bf16_t *>(a.out) + r * a.d + n;
          yr[0] = f32_to_bf16(acc[mi][0][q]);
          yr[16] = f32_to_bf16(acc[mi][1][q]);
        } else {
          float *pr = sa.part0 + (static_cast<size_t>(s) * sa.rows_cap + r) * a.d + n;
          pr[0] = acc[mi][0][q];
          pr[16] = acc[mi][1][q];
        }
      }
    }
}

// one wave per work item; item = ((grp * splits) + s) * nN + nb
template <bool GATEUP>
__global__ __launch_bounds__(256) void skinny_gemm_kernel(SkinnyArgs sa) {
  const GemmArgs &a = sa.g;
  const int nN = GATEUP ? a.m / 16 : a.d / 32;
  const long item = static_cast<long>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int nb = static_cast<int>(item % nN);
  const long rest = item / nN;
  const int s = static_cast<int>(rest % sa.splits);
  const int grp = static_cast<int>(rest / sa.splits);
  if (grp >= a.max_groups) return;
  const TileInfo ti = skinny_tile(a, grp);
  if (!ti.valid) return;
  const int blocks = (ti.rows + 15) >> 4;
  if (blocks <= 1)
    skinny_item<GATEUP, 1>(sa, ti, nb, s);
  else if (blocks <= 2)
    skinny_item<GATEUP, 2>(sa, ti, nb, s);
  else
    skinny_item<GATEUP, 4>(sa, ti, nb, s);
}

// H = SiLU(sum_s gate partials) * (sum_s up partials), splits added in order
__global__ __launch_bounds__(256) void swiglu_reduce_kernel(SkinnyArgs sa, const int32_t *n_rows) {
  const GemmArgs &a = sa.g;
  const int rows = a.dense_rows > 0 ? a.dense_rows : n_rows[0];
  const size_t total = static_cast<size_t>(rows) * a.m;
  bf16_t *H = static_cast<bf16_t *>(a.out);
  const size_t plane = static_cast<size_t>(sa.rows_cap) * a.m;
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < total;
       i += static_cast<size_t>(gridDim.x) * blockDim.x) {
    float gs = 0.f, us = 0.f;
    for (int s = 0; s < sa.splits; ++s) {
      gs += sa.part0[s * plane + i];
      us += sa.part1[s * plane + i];
    }
    H[i] = f32_to_bf16(silu(gs) * us);
  }
}

}  // namespace

hipError_t launch_skinny(const SkinnyArgs &sa, bool gateup, const int32_t *n_rows, hipStream_t stream) {
  const GemmArgs &a = sa.g;
  if (a.max_groups <= 0) return hipSuccess;
  const long nN = gateup ? a.m / 16 : a.d / 32;
  const long items = static_cast<long>(a.max_groups) * sa.splits * nN;
  const dim3 grid(static_cast<unsigned>((items + 3) / 4));
  if (gateup) {
    skinny_gemm_kernel<true><<<grid, 256, 0, stream>>>(sa);
    if (sa.splits > 1) {
      const size_t total = static_cast<size_t>(sa.rows_cap) * a.m;
      size_t blocks = (total + 255) / 256;
      if (blocks > 2048) blocks = 2048;
      swiglu_reduce_kernel<<<dim3(static_cast<unsigned>(blocks)), 256, 0, stream>>>(sa, n_rows);
    }
  } else {
    skinny_gemm_kernel<false><<<grid, 256, 0, stream>>>(sa);
  }
  return hipGetLastError();
}

}  // namespace ace
