// Grouped expert GEMMs of the sparsified MoE output (Eq. ace_sparse_output):
// every kept slot (token t, expert e) evaluates the SwiGLU expert of
// Eq. swiglu_expert, f_e(x) = W_down (SiLU(W_gate x) * (W_up x)), in nn.Linear
// layouts.  Rows are the compacted kept slots of the dispatch plan, grouped by
// expert, so every M tile multiplies rows of one expert against that expert's
// weights.
//
//   gateup: H[r, :] = SiLU(x_in[perm[r]] W_gate[e]^T) * (x_in[perm[r]] W_up[e]^T)
//           (the A rows are gathered through perm while staging the tile;
//           SiLU and the product are fused into the epilogue)
//   down:   Y[r, :] = H[r, :] W_down[e]^T
//
// bf16 path: bf16 MFMA (v_mfma_f32_16x16x32_bf16) with fp32 accumulation, tiles
// staged through LDS with double buffering (one barrier per K step), padded LDS
// rows (144 B) so the 16 rows an MFMA operand read touches hit distinct banks.
// fp32 path: plain tiled FMA (small parity workloads).
//
// Launch order is XCD-aware: workgroups are dealt to the 8 XCDs round-robin, so
// block b runs on XCD b % 8; the N tiles of one M tile are mapped to one XCD so
// the gathered activation rows they share stay in that XCD's L2.
#include "ace_internal.h"

namespace ace {

namespace {

constexpr int BK = 64;        // K step
constexpr int LDS_ROW = BK + 8;  // padded LDS row in elements (bf16: 144 B)
constexpr int GU_BN = 64;     // gate/up: intermediate features per tile (x2 weight rows)
constexpr int DN_BN = 128;    // down: output columns per tile

struct TileInfo {
  int e, row0, rows;
  bool valid;
};

__device__ __forceinline__ void map_block(int b, int nN, int *grp, int *nt) {
  const int xcd = b & 7;
  const int j = b >> 3;
  *grp = xcd + 8 * (j / nN);
  *nt = j % nN;
}

__device__ __forceinline__ TileInfo tile_info(const GemmArgs &a, int grp) {
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

__device__ __forceinline__ f32x4_t mfma_bf16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float silu(float v) { return v / (1.0f + expf(-v)); }

// stage 4 16-byte chunks of the A tile and 4 of the B tile.  A-tile rows past
// the tile's row count read the last valid row instead: every output row depends
// only on its own A row and those rows are never stored.
__device__ __forceinline__ void gload4(uint4 (&ra)[4], uint4 (&rb)[4], const bf16_t *const (&asrc)[4],
                                       const bf16_t *const (&bsrc)[4], int k0) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = *reinterpret_cast<const uint4 *>(asrc[i] + k0);
    rb[i] = *reinterpret_cast<const uint4 *>(bsrc[i] + k0);
  }
}

__device__ __forceinline__ void sstore4(bf16_t *as, bf16_t *bs, const uint4 (&ra)[4], const uint4 (&rb)[4],
                                        const int (&loff)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<uint4 *>(as + loff[i]) = ra[i];
    *reinterpret_cast<uint4 *>(bs + loff[i]) = rb[i];
  }
}

// one BK step of the gate/up tile from LDS: wave (wm, wn) owns 64 rows x 32 features
__device__ __forceinline__ void gateup_step(const bf16_t *As, const bf16_t *Bs, int wm, int wn, int r16, int kg,
                                            f32x4_t (&accg)[4][2], f32x4_t (&accu)[4][2]) {
#pragma unroll
  for (int kk = 0; kk < BK; kk += 32) {
    bf16x8_t af[4], bg[2], bu[2];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
      af[mi] = *reinterpret_cast<const bf16x8_t *>(&As[(wm * 64 + mi * 16 + r16) * LDS_ROW + kk + kg]);
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      bg[ni] = *reinterpret_cast<const bf16x8_t *>(&Bs[(wn * 32 + ni * 16 + r16) * LDS_ROW + kk + kg]);
      bu[ni] = *reinterpret_cast<const bf16x8_t *>(&Bs[(GU_BN + wn * 32 + ni * 16 + r16) * LDS_ROW + kk + kg]);
    }
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        accg[mi][ni] = mfma_bf16(af[mi], bg[ni], accg[mi][ni]);
        accu[mi][ni] = mfma_bf16(af[mi], bu[ni], accu[mi][ni]);
      }
  }
}

// one BK step of the down tile from LDS: wave (wm, wn) owns 64 rows x 64 columns
__device__ __forceinline__ void down_step(const bf16_t *As, const bf16_t *Bs, int wm, int wn, int r16, int kg,
                                          f32x4_t (&acc)[4][4]) {
#pragma unroll
  for (int kk = 0; kk < BK; kk += 32) {
    bf16x8_t af[4], bf[4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
      af[mi] = *reinterpret_cast<const bf16x8_t *>(&As[(wm * 64 + mi * 16 + r16) * LDS_ROW + kk + kg]);
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
      bf[ni] = *reinterpret_cast<const bf16x8_t *>(&Bs[(wn * 64 + ni * 16 + r16) * LDS_ROW + kk + kg]);
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = mfma_bf16(af[mi], bf[ni], acc[mi][ni]);
  }
}

// ------------------------------------------------------------------ bf16 gate/up
__global__ __launch_bounds__(256) void gateup_bf16_kernel(GemmArgs a) {
  const int nN = a.m / GU_BN;
  int grp, nt;
  map_block(blockIdx.x, nN, &grp, &nt);
  const TileInfo ti = tile_info(a, grp);
  if (!ti.valid) return;

  __shared__ __align__(16) bf16_t As[2][kTileM * LDS_ROW];
  __shared__ __align__(16) bf16_t Bs[2][2 * GU_BN * LDS_ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, m = a.m;
  const int f0 = nt * GU_BN;
  const bf16_t *xn = static_cast<const bf16_t *>(a.act);
  const bf16_t *wg = static_cast<const bf16_t *>(a.w0);
  const bf16_t *wu = static_cast<const bf16_t *>(a.w1);

  // each thread stages 4 16-byte chunks of the A tile and 4 of the B tile per K step
  const bf16_t *asrc[4];
  const bf16_t *bsrc[4];
  int loff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int r = c >> 3, c8 = c & 7;
    loff[i] = r * LDS_ROW + c8 * 8;
    const int rr = min(r, ti.rows - 1);
    const int tok = a.perm ? a.perm[ti.row0 + rr] : ti.row0 + rr;
    asrc[i] = xn + static_cast<size_t>(tok) * d + c8 * 8;
    const bf16_t *w = (r < GU_BN) ? wg : wu;
    bsrc[i] = w + (static_cast<size_t>(ti.e) * m + f0 + (r & (GU_BN - 1))) * d + c8 * 8;
  }
  uint4 ra[4], rb[4];
  const int wm = wave >> 1, wn = wave & 1;
  const int r16 = lane & 15, kg = (lane >> 4) * 8;
  f32x4_t accg[4][2], accu[4][2];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      accg[mi][ni] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      accu[mi][ni] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

  const int nk = d / BK;
  gload4(ra, rb, asrc, bsrc, 0);
  sstore4(As[0], Bs[0], ra, rb, loff);
  __syncthreads();
  for (int kt = 0; kt < nk - 1; ++kt) {
    const int buf = kt & 1;
    gload4(ra, rb, asrc, bsrc, (kt + 1) * BK);
    gateup_step(As[buf], Bs[buf], wm, wn, r16, kg, accg, accu);
    sstore4(As[buf ^ 1], Bs[buf ^ 1], ra, rb, loff);
    __syncthreads();
  }
  gateup_step(As[(nk - 1) & 1], Bs[(nk - 1) & 1], wm, wn, r16, kg, accg, accu);

  bf16_t *H = static_cast<bf16_t *>(a.out);
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * 64 + mi * 16 + (lane >> 4) * 4 + i;
        const int f = f0 + wn * 32 + ni * 16 + r16;
        if (r < ti.rows) {
          const float h = silu(accg[mi][ni][i]) * accu[mi][ni][i];
          H[static_cast<size_t>(ti.row0 + r) * m + f] = f32_to_bf16(h);
        }
      }
}

// ------------------------------------------------------------------ bf16 down
__global__ __launch_bounds__(256) void down_bf16_kernel(GemmArgs a) {
  const int nN = a.d / DN_BN;
  int grp, nt;
  map_block(blockIdx.x, nN, &grp, &nt);
  const TileInfo ti = tile_info(a, grp);
  if (!ti.valid) return;

  __shared__ __align__(16) bf16_t As[2][kTileM * LDS_ROW];
  __shared__ __align__(16) bf16_t Bs[2][DN_BN * LDS_ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, m = a.m;
  const int n0 = nt * DN_BN;
  const bf16_t *H = static_cast<const bf16_t *>(a.act);
  const bf16_t *wd = static_cast<const bf16_t *>(a.w0);

  const bf16_t *asrc[4];
  const bf16_t *bsrc[4];
  int loff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int r = c >> 3, c8 = c & 7;
    loff[i] = r * LDS_ROW + c8 * 8;
    asrc[i] = H + static_cast<size_t>(ti.row0 + min(r, ti.rows - 1)) * m + c8 * 8;
    bsrc[i] = wd + (static_cast<size_t>(ti.e) * d + n0 + r) * m + c8 * 8;
  }

  uint4 ra[4], rb[4];

  const int wm = wave >> 1, wn = wave & 1;
  const int r16 = lane & 15, kg = (lane >> 4) * 8;
  f32x4_t acc[4][4];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = m / BK;
  gload4(ra, rb, asrc, bsrc, 0);
  sstore4(As[0], Bs[0], ra, rb, loff);
  __syncthreads();
  for (int kt = 0; kt < nk - 1; ++kt) {
    const int buf = kt & 1;
    gload4(ra, rb, asrc, bsrc, (kt + 1) * BK);
    down_step(As[buf], Bs[buf], wm, wn, r16, kg, acc);
    sstore4(As[buf ^ 1], Bs[buf ^ 1], ra, rb, loff);
    __syncthreads();
  }
  down_step(As[(nk - 1) & 1], Bs[(nk - 1) & 1], wm, wn, r16, kg, acc);

  bf16_t *Y = static_cast<bf16_t *>(a.out);
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * 64 + mi * 16 + (lane >> 4) * 4 + i;
        const int n = n0 + wn * 64 + ni * 16 + r16;
        if (r < ti.rows) Y[static_cast<size_t>(ti.row0 + r) * d + n] = f32_to_bf16(acc[mi][ni][i]);
      }
}

// ------------------------------------------------------------------ fp32 (tiled FMA)
constexpr int F_BN = 16;
constexpr int F_BK = 16;

__global__ __launch_bounds__(256) void gateup_f32_kernel(GemmArgs a) {
  const int nN = a.m / F_BN;
  int grp, nt;
  map_block(blockIdx.x, nN, &grp, &nt);
  const TileInfo ti = tile_info(a, grp);
  if (!ti.valid) return;
  __shared__ float As[kTileM][F_BK + 1];
  __shared__ float Bg[F_BN][F_BK + 1];
  __shared__ float Bu[F_BN][F_BK + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int d = a.d, m = a.m, f0 = nt * F_BN;
  const float *xn = static_cast<const float *>(a.act);
  const float *wg = static_cast<const float *>(a.w0);
  const float *wu = static_cast<const float *>(a.w1);
  int tok[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = (tid + 256 * j) >> 4;
    tok[j] = (r < ti.rows) ? (a.perm ? a.perm[ti.row0 + r] : ti.row0 + r) : -1;
  }
  float ag[8] = {0}, au[8] = {0};
  for (int k0 = 0; k0 < d; k0 += F_BK) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = tid + 256 * j;
      const int r = c >> 4, kk = c & 15;
      As[r][kk] = (tok[j] >= 0) ? xn[static_cast<size_t>(tok[j]) * d + k0 + kk] : 0.f;
    }
    {
      const int r = tid >> 4, kk = tid & 15;
      const size_t wrow = (static_cast<size_t>(ti.e) * m + f0 + r) * d + k0 + kk;
      Bg[r][kk] = wg[wrow];
      Bu[r][kk] = wu[wrow];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < F_BK; ++kk) {
      const float bgv = Bg[tx][kk], buv = Bu[tx][kk];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ag[i] = fmaf(As[ty + 16 * i][kk], bgv, ag[i]);
        au[i] = fmaf(As[ty + 16 * i][kk], buv, au[i]);
      }
    }
    __syncthreads();
  }
  float *H = static_cast<float *>(a.out);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = ty + 16 * i;
    if (r < ti.rows) H[static_cast<size_t>(ti.row0 + r) * m + f0 + tx] = silu(ag[i]) * au[i];
  }
}

__global__ __launch_bounds__(256) void down_f32_kernel(GemmArgs a) {
  const int nN = a.d / F_BN;
  int grp, nt;
  map_block(blockIdx.x, nN, &grp, &nt);
  const TileInfo ti = tile_info(a, grp);
  if (!ti.valid) return;
  __shared__ float As[kTileM][F_BK + 1];
  __shared__ float Bs[F_BN][F_BK + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int d = a.d, m = a.m, n0 = nt * F_BN;
  const float *H = static_cast<const float *>(a.act);
  const float *wd = static_cast<const float *>(a.w0);
  float acc[8] = {0};
  for (int k0 = 0; k0 < m; k0 += F_BK) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = tid + 256 * j;
      const int r = c >> 4, kk = c & 15;
      As[r][kk] = (r < ti.rows) ? H[static_cast<size_t>(ti.row0 + r) * m + k0 + kk] : 0.f;
    }
    {
      const int r = tid >> 4, kk = tid & 15;
      Bs[r][kk] = wd[(static_cast<size_t>(ti.e) * d + n0 + r) * m + k0 + kk];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < F_BK; ++kk) {
      const float bv = Bs[tx][kk];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = fmaf(As[ty + 16 * i][kk], bv, acc[i]);
    }
    __syncthreads();
  }
  float *Y = static_cast<float *>(a.out);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = ty + 16 * i;
    if (r < ti.rows) Y[static_cast<size_t>(ti.row0 + r) * d + n0 + tx] = acc[i];
  }
}

unsigned grid_for(int max_groups, int nN) {
  const int g8 = (max_groups + 7) / 8;
  return static_cast<unsigned>(8 * nN * g8);
}

}  // namespace

hipError_t launch_gateup(const GemmArgs &a, bool bf16, hipStream_t stream) {
  if (a.max_groups <= 0) return hipSuccess;
  if (bf16)
    gateup_bf16_kernel<<<dim3(grid_for(a.max_groups, a.m / GU_BN)), 256, 0, stream>>>(a);
  else
    gateup_f32_kernel<<<dim3(grid_for(a.max_groups, a.m / F_BN)), 256, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_down(const GemmArgs &a, bool bf16, hipStream_t stream) {
  if (a.max_groups <= 0) return hipSuccess;
  if (bf16)
    down_bf16_kernel<<<dim3(grid_for(a.max_groups, a.d / DN_BN)), 256, 0, stream>>>(a);
  else
    down_f32_kernel<<<dim3(grid_for(a.max_groups, a.d / F_BN)), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
