// Grouped expert GEMMs for small batches (decode): at most 64 tokens, so every
// expert has at most 64 kept rows and the layer is a batch of weight-streaming
// GEMVs.  Work is split so that thousands of waves stream weights at once:
//  * a work item is one wave: one tile (expert) x 16 features (gate/up: a gate
//    block and an up block) or 32 output columns (down) x one K split;
//  * the wave streams its weight rows and its activation rows into a private
//    LDS ring with global_load_lds_dwordx4, one 8-row x 128-byte unit per
//    instruction (whole cache lines; see lds_dma.h; weights carry the
//    non-temporal hint when the wave makes one pass over them), P stages of 64 k
//    deep, and waits only on its own vmcnt: no barriers, waves run independently;
//  * it reads MFMA fragments back from the ring and multiplies them with
//    v_mfma_f32_16x16x32_bf16;
//  * with one K split the epilogue writes H (SwiGLU applied) or Y in bf16;
//    gate/up with several splits runs the splits of one 16-feature block as the
//    waves of one workgroup, which add their fp32 partial sums in split order
//    through LDS and write H (no reduction kernel); down with several splits
//    writes fp32 partial sums, which the combine kernel adds in split order, so
//    results do not depend on scheduling;
//  * batches of 2-4 router chunks need no plan kernel: each gate/up wave derives
//    its tile and the tokens of its rows from the router's per-chunk counts and
//    the routing (self_tile), and the gate/up launch writes the plan outputs and
//    the tile list for the down launch.
#include "lds_dma.h"

namespace ace {

namespace {

struct TileInfo {
  int e, row0, rows;
  bool valid;
};

// Tile grp of the dispatch plan derived by this wave (SkinnyArgs::self_plan).
// Lane l holds experts 4l .. 4l+3: their kept-slot counts (summed over the G
// chunks) give, by wave scans, the experts with kept slots in id order (tile
// grp is the grp-th of them) and their row offsets.  Lane t (t < T <= 64) finds
// the slot of token t routed to the tile's expert, if kept; ranks in token
// order give the rows, and lane r receives the token of row r (*tok).  The same
// integers as the plan kernels: rows in (expert, token) order.
__device__ TileInfo self_tile(const SkinnyArgs &sa, int grp, bool write_slots, bool write_plan, int *tok) {
  const int lane = threadIdx.x & 63;
  const int N = sa.N;
  // routing of token `lane` (issued first: independent of the counts)
  int te[kMaxK];
  uint8_t tk[kMaxK];
#pragma unroll
  for (int i = 0; i < kMaxK; ++i) {
    const bool in = lane < sa.T && i < sa.k;
    const size_t o = static_cast<size_t>(lane) * sa.k + i;
    te[i] = in ? sa.topk_idx[o] : -1;
    tk[i] = in ? sa.keep[o] : 0;
  }
  int c[4] = {0, 0, 0, 0};
  if ((N & 3) == 0) {
    // four experts per 32-bit word (rows of N bytes stay 4-byte aligned)
    for (int g = 0; g < sa.G; ++g) {
      const uint32_t w = 4 * lane < N ? reinterpret_cast<const uint32_t *>(sa.chunk_count + static_cast<size_t>(g) * N)[lane] : 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] += (w >> (8 * j)) & 0xFFu;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = 4 * lane + j;
      for (int g = 0; g < sa.G; ++g) c[j] += e < N ? sa.chunk_count[static_cast<size_t>(g) * N + e] : 0;
    }
  }
  const int na = (c[0] > 0) + (c[1] > 0) + (c[2] > 0) + (c[3] > 0);
  const int ns = c[0] + c[1] + c[2] + c[3];
  int na_inc = na, ns_inc = ns;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int va = __shfl_up(na_inc, o), vs = __shfl_up(ns_inc, o);
    if (lane >= o) {
      na_inc += va;
      ns_inc += vs;
    }
  }
  const int na_ex = na_inc - na, ns_ex = ns_inc - ns;
  const int n_active = __shfl(na_inc, 63);
  if (write_plan) {
    int off = ns_ex, a_idx = na_ex;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = 4 * lane + j;
      if (e < N) {
        sa.counts[e] = c[j];
        sa.offsets[e] = off;
        if (c[j] > 0) {
          sa.tile_expert[a_idx] = e;
          sa.tile_row0[a_idx] = off;
          sa.tile_rows[a_idx] = c[j];
          ++a_idx;
        }
      }
      off += c[j];
    }
    if (lane == 63) {
      sa.offsets[N] = ns_inc;
      sa.n_tiles[0] = n_active;
    }
  }
  TileInfo ti;
  ti.valid = grp < n_active;
  if (!ti.valid) {
    ti.e = ti.row0 = ti.rows = 0;
    *tok = 0;
    return ti;
  }
  // the lane holding tile grp's expert, then the expert among its four
  const unsigned long long owner = __ballot(na_ex <= grp && grp < na_inc);
  const int L = __ffsll(static_cast<long long>(owner)) - 1;
  int e_l = 0, r0_l = ns_ex, rows_l = 0, q = grp - na_ex, found = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (!found && c[j] > 0) {
      if (q == 0) {
        e_l = 4 * lane + j;
        rows_l = c[j];
        found = 1;
      } else {
        --q;
        r0_l += c[j];
      }
    } else if (!found) {
      r0_l += c[j];
    }
  }
  ti.e = __shfl(e_l, L);
  ti.row0 = __shfl(r0_l, L);
  ti.rows = __shfl(rows_l, L);
  // tokens of the tile's rows
  int slot = -1;
#pragma unroll
  for (int i = 0; i < kMaxK; ++i)
    if (te[i] == ti.e && tk[i]) slot = i;
  const bool hit = slot >= 0;
  const unsigned long long hits = __ballot(hit);
  const int rank = __popcll(hits & ((1ull << lane) - 1ull));
  // a permutation of the 64 lanes (hits to 0 .. n-1 in token order, the others
  // after them), so every lane receives exactly one value: lane r <- token of row r
  const int dst = hit ? rank : __popcll(hits) + (lane - rank);
  *tok = __builtin_amdgcn_ds_permute(dst << 2, lane);
  if (write_slots && hit) {
    const int row = ti.row0 + rank;
    sa.slot_row[static_cast<size_t>(lane) * sa.k + slot] = row;
    sa.perm[row] = lane;
  }
  return ti;
}

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

constexpr int kSkinnyWavesPerGroup = 4;
constexpr int kSkinnyRingBytes = 20 * 1024;  // LDS ring of one wave (4 waves: 80 KB, two workgroups per CU)

// ring geometry for AU activation units per stage: a stage holds 4 weight units
// (2 blocks x 2 row halves) then the activation units (2 per 16-row block, or
// just one when the tile has at most 8 rows)
template <int AU> struct SkinnyRing {
  static constexpr int NU = 4 + AU;                                    // units (DMAs) per stage
  static constexpr int STAGE = NU * kUnitBytes;
  static constexpr int P = kSkinnyRingBytes / STAGE;                   // stages in the ring
  static_assert(P >= 2, "ring too shallow");
  static_assert((P - 1) * NU <= 63, "outstanding DMAs exceed the wait table");
};

// whether a ring holds two stages of a 32-row (two-block) item
constexpr bool kSkinnyTwoBlocks = kSkinnyRingBytes / ((4 + 4) * kUnitBytes) >= 2;

// red != null (gate/up, K splits as the waves of one workgroup, wave index =
// split): the partial sums go through red (LDS, over the workgroup's rings) and
// wave 0 adds them in split order and writes H; every wave of the workgroup
// calls this with the same tile rows.
template <bool GATEUP, int MB, int AU>
__device__ __forceinline__ void skinny_item(const SkinnyArgs &sa, const TileInfo &ti, int nb, int s, int rot,
                                            bool once, int tok, int rbase, uint8_t *ring, f32x4_t *red) {
  static_assert(AU == 2 * MB || (MB == 1 && AU == 1), "activation units cover the row blocks");
  using R = SkinnyRing<AU>;
  constexpr int P = R::P, NU = R::NU;
  const GemmArgs &a = sa.g;
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const int ur = lane >> 3;  // DMA lane -> row in its unit
  const int K = GATEUP ? a.d : a.m;
  const int kc = K / sa.splits;
  const int kbase = s * kc;
  const int nk = kc / 64;

  // weight units t = 2 cb + j: block cb (gate/up: gate, up; down: 16-column halves), row half j
  const bf16_t *src[NU];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int cb = t >> 1, j = t & 1;
    const int c = kbase + 8 * unit_chunk(lane);
    if (GATEUP) {
      const size_t f = static_cast<size_t>(ti.e) * a.m + nb * 16 + 8 * j + ur;
      src[t] = static_cast<const bf16_t *>(cb ? a.w1 : a.w0) + f * a.d + c;
    } else {
      const size_t n = static_cast<size_t>(ti.e) * a.d + nb * 32 + cb * 16 + 8 * j + ur;
      src[t] = static_cast<const bf16_t *>(a.w0) + n * a.m + c;
    }
  }
  // activation units 4 + 2 mi + j: row block mi, row half j (AU == 1: rows 0-7 only)
  const bf16_t *act = static_cast<const bf16_t *>(a.act);
#pragma unroll
  for (int t = 4; t < NU; ++t) {
    const int mi = (t - 4) >> 1, j = t & 1;
    const int row = min(mi * 16 + 8 * j + ur, ti.rows - 1);  // rows past the tile repeat its last row
    // self_plan: the token of tile row r sits in lane r of tok (tile rows <= 64;
    // this item covers tile rows rbase ..)
    const int src_row = sa.self_plan ? __shfl(tok, rbase + row) : a.perm ? a.perm[ti.row0 + row] : ti.row0 + row;
    src[t] = act + static_cast<size_t>(src_row) * K + kbase + 8 * unit_chunk(lane);
  }
  const uint32_t ring_lds = lds_addr(ring);
  // Stage st covers the 64-wide K block (st + k0) % nk of this split: waves start
  // at different K blocks, so rows 4 KB apart are not all read at one offset at
  // once (that concentrates the stream on a few HBM channels).
  const int k0 = rot % nk;
  // stage st -> slot st % P; its units at slot * STAGE + t * kUnitBytes
  auto issue = [&](int st) {
    const uint32_t base = ring_lds + (st % P) * R::STAGE;
    const int kb = st + k0 < nk ? st + k0 : st + k0 - nk;
    // weights: non-temporal when this is the item's only pass over them
    if (once) {
#pragma unroll
      for (int t = 0; t < 4; ++t) dma16_stream(src[t] + kb * 64, base + t * kUnitBytes);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) dma16(src[t] + kb * 64, base + t * kUnitBytes);
    }
#pragma unroll
    for (int t = 4; t < NU; ++t) dma16(src[t] + kb * 64, base + t * kUnitBytes);  // activation rows
  };

  f32x4_t acc[MB][2];
#pragma unroll
  for (int mi = 0; mi < MB; ++mi) {
    acc[mi][0] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    acc[mi][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }
  const int rd0 = unit_read_offset(lane, 0), rd1 = unit_read_offset(lane, 1);
  // with one activation unit, lanes of rows 8-15 (past the tile) read inside that unit
  const int ra0 = (AU == 1 && (lane & 8)) ? rd0 - kUnitBytes : rd0;
  const int ra1 = (AU == 1 && (lane & 8)) ? rd1 - kUnitBytes : rd1;
  for (int st = 0; st < P - 1 && st < nk; ++st) issue(st);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + P - 1 < nk) {
      // the slot it refills held stage kt-1, whose LDS reads this wave issued last iteration
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      issue(kt + P - 1);
    }
    wait_vmcnt(NU * min(P - 1, nk - 1 - kt));  // stage kt landed
    const uint8_t *sl = ring + (kt % P) * R::STAGE;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int rd = h ? rd1 : rd0, ra = h ? ra1 : ra0;
      bf16x8_t bf[2];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
        bf[cb] = *reinterpret_cast<const bf16x8_t *>(sl + cb * 2 * kUnitBytes + rd);
#pragma unroll
      for (int mi = 0; mi < MB; ++mi) {
        const bf16x8_t av = *reinterpret_cast<const bf16x8_t *>(sl + (4 + 2 * mi) * kUnitBytes + ra);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[mi][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bf[cb], acc[mi][cb], 0, 0, 0);
      }
    }
  }

  if (GATEUP && red != nullptr) {
    // every wave's last wait covered all its DMAs, so after the barrier no ring
    // is written any more and red may overlay them
    __syncthreads();
    const int w = threadIdx.x >> 6;
#pragma unroll
    for (int mi = 0; mi < MB; ++mi)
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) red[((w * MB + mi) * 2 + cb) * 64 + lane] = acc[mi][cb];
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int mi = 0; mi < MB; ++mi)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // the splits in order from zero, as a separate reduction would add them
          float gs = 0.f, us = 0.f;
          for (int sp = 0; sp < sa.splits; ++sp) {
            gs += red[((sp * MB + mi) * 2 + 0) * 64 + lane][q];
            us += red[((sp * MB + mi) * 2 + 1) * 64 + lane][q];
          }
          const int row = mi * 16 + 4 * g + q;
          if (row < ti.rows)
            static_cast<bf16_t *>(a.out)[static_cast<size_t>(ti.row0 + row) * a.m + nb * 16 + r16] =
                f32_to_bf16(silu_for_bf16(gs) * us);
        }
    }
    __syncthreads();  // red is overwritten by the next pass's DMAs
    return;
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
          static_cast<bf16_t *>(a.out)[r * a.m + f] = f32_to_bf16(silu_for_bf16(acc[mi][0][q]) * acc[mi][1][q]);
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

// WGS = 0: one wave per work item, item = ((grp * splits) + s) * nN + nb, four
// independent waves per workgroup.  WGS = splits (gate/up): workgroup
// grp * nN + nb, wave s; the waves add their partial sums through LDS.
template <bool GATEUP, int WGS>
__global__ __launch_bounds__((WGS ? WGS : kSkinnyWavesPerGroup) * 64) void skinny_gemm_kernel(SkinnyArgs sa) {
  constexpr int NW = WGS ? WGS : kSkinnyWavesPerGroup;
  static_assert(!WGS || GATEUP, "workgroup reduction: gate/up only");
  static_assert(!WGS || 2 * 2 * 64 * 16 <= kSkinnyRingBytes, "partials of a wave fit its ring");
  __shared__ __align__(16) uint8_t smem[NW * kSkinnyRingBytes];
  const GemmArgs &a = sa.g;
  const int nN = GATEUP ? a.m / 16 : a.d / 32;
  const int wave = threadIdx.x >> 6;
  uint8_t *ring = smem + wave * kSkinnyRingBytes;
  f32x4_t *red = WGS ? reinterpret_cast<f32x4_t *>(smem) : nullptr;
  const long item = static_cast<long>(blockIdx.x) * NW + wave;
  int nb, s, grp;
  if constexpr (WGS > 0) {
    nb = static_cast<int>(blockIdx.x % nN);
    grp = static_cast<int>(blockIdx.x / nN);
    s = wave;
  } else {
    nb = static_cast<int>(item % nN);
    const long rest = item / nN;
    s = static_cast<int>(rest % sa.splits);
    grp = static_cast<int>(rest / sa.splits);
  }
  if (grp >= a.max_groups) return;
  int tok = 0;
  const TileInfo ti = (GATEUP && sa.self_plan) ? self_tile(sa, grp, nb == 0 && s == 0, item == 0, &tok)
                                              : skinny_tile(a, grp);
  if (!ti.valid) return;
  const int blocks = (ti.rows + 15) >> 4;
  const int rot = static_cast<int>(item & 0x7fffffff);
  if (ti.rows <= 8) {
    skinny_item<GATEUP, 1, 1>(sa, ti, nb, s, rot, true, tok, 0, ring, red);
  } else if (blocks <= 1 || !kSkinnyTwoBlocks) {
    // 16 rows per pass (more than 16 rows re-read the weights, mostly from L2)
    for (int r = 0; r < ti.rows; r += 16) {
      TileInfo part = ti;
      part.row0 = ti.row0 + r;
      part.rows = min(16, ti.rows - r);
      skinny_item<GATEUP, 1, 2>(sa, part, nb, s, rot, ti.rows <= 16, tok, r, ring, red);
    }
  } else if constexpr (kSkinnyTwoBlocks) {
    // 32 rows per pass
    for (int r = 0; r < ti.rows; r += 32) {
      TileInfo part = ti;
      part.row0 = ti.row0 + r;
      part.rows = min(32, ti.rows - r);
      skinny_item<GATEUP, 2, 4>(sa, part, nb, s, rot, ti.rows <= 32, tok, r, ring, red);
    }
  }
}

constexpr int kMaxGateUpSplits = 8;  // K splits of the small-batch gate/up GEMM

// H = SiLU(sum_s gate partials) * (sum_s up partials), splits added in order.
// All splits' partials are loaded before the first add, so the L2 round trips
// overlap instead of following one another; the sums keep split order.
__global__ __launch_bounds__(256) void swiglu_reduce_kernel(SkinnyArgs sa, const int32_t *n_rows) {
  const GemmArgs &a = sa.g;
  const int rows = a.dense_rows > 0 ? a.dense_rows : n_rows[0];
  const size_t total = static_cast<size_t>(rows) * a.m;
  bf16_t *H = static_cast<bf16_t *>(a.out);
  const size_t plane = static_cast<size_t>(sa.rows_cap) * a.m;
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < total;
       i += static_cast<size_t>(gridDim.x) * blockDim.x) {
    float pg[kMaxGateUpSplits], pu[kMaxGateUpSplits];
#pragma unroll
    for (int s = 0; s < kMaxGateUpSplits; ++s)
      if (s < sa.splits) {
        pg[s] = sa.part0[s * plane + i];
        pu[s] = sa.part1[s * plane + i];
      }
    float gs = 0.f, us = 0.f;
#pragma unroll
    for (int s = 0; s < kMaxGateUpSplits; ++s) {
      if (s >= sa.splits) break;
      gs += pg[s];
      us += pu[s];
    }
    H[i] = f32_to_bf16(silu_for_bf16(gs) * us);
  }
}

}  // namespace

hipError_t launch_skinny(const SkinnyArgs &sa, bool gateup, const int32_t *n_rows, hipStream_t stream) {
  const GemmArgs &a = sa.g;
  if (a.max_groups <= 0) return hipSuccess;
  const long nN = gateup ? a.m / 16 : a.d / 32;
  const long items = static_cast<long>(a.max_groups) * sa.splits * nN;
  const dim3 grid(static_cast<unsigned>((items + kSkinnyWavesPerGroup - 1) / kSkinnyWavesPerGroup));
  if (gateup) {
    if (sa.splits > kMaxGateUpSplits) return hipErrorInvalidValue;
    // several K splits: the splits of a 16-feature block are one workgroup's waves
    const dim3 wg_grid(static_cast<unsigned>(static_cast<long>(a.max_groups) * nN));
    switch (sa.splits) {
      case 1: skinny_gemm_kernel<true, 0><<<grid, kSkinnyWavesPerGroup * 64, 0, stream>>>(sa); break;
      case 2: skinny_gemm_kernel<true, 2><<<wg_grid, 2 * 64, 0, stream>>>(sa); break;
      case 4: skinny_gemm_kernel<true, 4><<<wg_grid, 4 * 64, 0, stream>>>(sa); break;
      case 8: skinny_gemm_kernel<true, 8><<<wg_grid, 8 * 64, 0, stream>>>(sa); break;
      default: {
        // other split counts: partial sums, then the reduction kernel
        skinny_gemm_kernel<true, 0><<<grid, kSkinnyWavesPerGroup * 64, 0, stream>>>(sa);
        const size_t total = static_cast<size_t>(sa.rows_cap) * a.m;
        size_t blocks = (total + 255) / 256;
        if (blocks > 2048) blocks = 2048;
        swiglu_reduce_kernel<<<dim3(static_cast<unsigned>(blocks)), 256, 0, stream>>>(sa, n_rows);
      }
    }
  } else {
    skinny_gemm_kernel<false, 0><<<grid, kSkinnyWavesPerGroup * 64, 0, stream>>>(sa);
  }
  return hipGetLastError();
}

}  // namespace ace
