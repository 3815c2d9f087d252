// Grouped expert GEMMs of the sparsified MoE output (Eq. ace_sparse_output):
// every kept slot (token t, expert e) evaluates the SwiGLU expert of
// Eq. swiglu_expert, f_e(x) = W_down (SiLU(W_gate x) * (W_up x)), in nn.Linear
// layouts.  Rows are the compacted kept slots of the dispatch plan, grouped by
// expert, so every M tile multiplies rows of one expert against that expert's
// weights.
//
//   gateup: H[r, :] = SiLU(x_in[perm[r]] W_gate[e]^T) * (x_in[perm[r]] W_up[e]^T)
//           (A rows gathered through perm; SiLU and the product fused into the
//           epilogue)
//   down:   Y[r, :] = H[r, :] W_down[e]^T
//
// bf16 path (MI355X, bf16 MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation).
// With 50% of 32768 slots kept over 128 experts an expert sees ~90-190 rows, so
// the layer streams every activated expert's weights once and is HBM-bound:
//  * an M tile holds up to 256 rows, so an expert's weights are read once per
//    tile (a 128-row tile would re-read them for every expert past 128 rows);
//    the row count selects one of four unrolled bodies (64..256 rows) so MFMAs
//    and loads are issued only for the 16-row blocks a tile has;
//  * operands move HBM/L2 -> LDS with global_load_lds_dwordx4 (no VGPR staging)
//    through two LDS rings in 160 KB: activations (L2-resident) 2-4 K stages deep,
//    expert weights (from HBM; with the non-temporal hint when no other M tile
//    reads them) 3-8 stages deep; each wave waits only for the
//    stage it computes next (vmcnt counted exactly from the issue schedule; with
//    two activation stages one of two constants, since a run-time count becomes a
//    branch tree that costs matrix-bound tiles several percent), then one barrier
//    per K step;
//  * one DMA instruction moves 8 rows x 128 bytes (whole cache lines) and lane i
//    lands at byte 16*i; the chunk a lane fetches is XOR-swizzled by its row so
//    the MFMA fragment reads (16 rows x 16 bytes) are bank-conflict free;
//  * 8 waves (two per SIMD, so one wave's LDS reads overlap the other's MFMAs)
//    as 4 x 2: a wave owns a quarter of the row blocks (interleaved, so short
//    tiles stay balanced) and two column groups (gate/up: gate and up blocks of
//    the same 16 features, so SwiGLU happens in registers; down: 32 columns);
//  * the down launch gives each workgroup two N tiles of one M tile, run as one
//    pipeline (the second tile's first stages load under the first's last steps).
// fp32 path: fp32 MFMA (v_mfma_f32_16x16x4f32) on LDS-staged operands (small
// parity workloads).
//
// Launch order is XCD-aware: workgroups are dealt to the 8 XCDs round-robin, so
// block b runs on XCD b % 8; the N tiles of one M tile are mapped to one XCD so
// the activation rows they share stay in that XCD's L2.
#include "gemm_pipe.h"
#include "lds_dma.h"

namespace ace {

namespace {

constexpr int kFragBytes = kUnitBytes;  // one staged unit (8 rows x 64 bf16, or 16 rows x 32)
constexpr int kLdsBytes = kPipeLdsBytes;
static_assert(kFragBytes == kPipeUnitBytes, "one DMA unit per fragment");

struct TileInfo {
  int e, row0, rows;
  bool valid;
  bool sh;    // a tile of the appended dense expert
  bool once;  // no other M tile of this launch reads this tile's expert weights
};

__device__ __forceinline__ void map_block(int b, int nN, int *grp, int *nt) {
  const int xcd = b & 7;
  const int j = b >> 3;
  *grp = xcd + 8 * (j / nN);
  *nt = j % nN;
}

__device__ __forceinline__ TileInfo tile_info(const GemmArgs &a, int grp) {
  TileInfo ti;
  ti.sh = false;
  if (a.dense_rows > 0) {
    ti.e = 0;
    ti.row0 = grp * kTileM;
    ti.rows = min(kTileM, a.dense_rows - ti.row0);
    ti.valid = ti.rows > 0;
    ti.once = a.dense_rows <= kTileM;
  } else {
    const int nr = a.n_tiles[0];
    if (a.tile_order && grp < nr) grp = a.tile_order[grp];
    ti.valid = grp < nr;
    ti.e = ti.valid ? a.tile_expert[grp] : 0;
    ti.row0 = ti.valid ? a.tile_row0[grp] : 0;
    ti.rows = ti.valid ? a.tile_rows[grp] : 0;
    // an expert's tiles are consecutive in the list
    ti.once = ti.valid && !(grp > 0 && a.tile_expert[grp - 1] == ti.e) &&
              !(grp + 1 < nr && a.tile_expert[grp + 1] == ti.e);
    if (!ti.valid && grp - nr < a.sh_tiles) {
      ti.sh = true;
      ti.e = 0;
      ti.row0 = (grp - nr) * kTileM;
      ti.rows = min(kTileM, a.sh_rows - ti.row0);
      ti.valid = ti.rows > 0;
      ti.once = a.sh_tiles == 1;
    }
  }
  return ti;
}

__device__ __forceinline__ float silu(float v) { return v / (1.0f + expf(-v)); }  // fp32 layers


constexpr int kGemmWaves = 8;  // waves per workgroup (two per SIMD)
// 32-wide k halves per pipeline stage.  Two (64-wide stages) measured faster than
// one with deeper rings: the stream rate, not the bytes in flight, is the limit.
template <int CG> constexpr int stage_halves() { return 2; }

// Pipe, cum_ops and pending_ok (gemm_pipe.h): ring depths per tile shape and
// the exact wait counts of a wave's DMA issue sequence.

// Output stores of gemm_tile: lane holds column r16 of each block, rows 4*g + q.
template <bool GATEUP, int MW, int CW, int RW, int BN>
__device__ __forceinline__ void store_tile_impl(const GemmArgs &a, const TileInfo &ti, void *outp,
                                                f32x4_t (&acc)[MW][2 * CW], int nt, int wr, int wc, int r16, int g) {
#pragma unroll
  for (int fl = 0; fl < CW; ++fl) {
    const int grp = wc * CW + fl;
    if (GATEUP) {
      bf16_t *H = static_cast<bf16_t *>(outp);
      const int f = nt * BN + grp * 16 + r16;
#pragma unroll
      for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = (wr + RW * i) * 16 + 4 * g + q;
          if (row < ti.rows)
            H[static_cast<size_t>(ti.row0 + row) * a.m + f] =
                f32_to_bf16(silu_for_bf16(acc[i][fl * 2][q]) * acc[i][fl * 2 + 1][q]);
        }
    } else {
      bf16_t *Y = static_cast<bf16_t *>(outp);
      const int n = nt * BN + grp * 32 + r16;
#pragma unroll
      for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = (wr + RW * i) * 16 + 4 * g + q;
          if (row < ti.rows) {
            bf16_t *yr = Y + static_cast<size_t>(ti.row0 + row) * a.d + n;
            yr[0] = f32_to_bf16(acc[i][fl * 2][q]);
            yr[16] = f32_to_bf16(acc[i][fl * 2 + 1][q]);
          }
        }
    }
  }
}

// One M tile x ntiles (1 or 2) consecutive N tiles from nt0, with MB 16-row
// blocks, CG column groups and KH = 2 k halves per stage (64-wide stages: 128
// bytes of every row).  One DMA
// instruction moves an 8-row unit: 8 rows x 128 bytes, each row a whole cache
// line (16-row x 64-byte fragments touch twice as many lines per instruction and
// stream measurably slower).  A stage of A holds units u = 2 rb + j (row block
// rb, row half j), wave w staging u = w, w+W, ...; a stage of B holds units
// b = 2 (2 fg + cb) + j (column group fg, block cb (gate/up: 0 gate, 1 up;
// down: the group's two 16-column halves), row half j), wave w staging
// b = w*NB .. w*NB+NB-1.  Inside a unit, row r's 16-byte chunk c sits in slot
// c ^ r (both units of a block alike), so the MFMA fragment reads (16 rows, one
// chunk each) run at the full LDS rate.  Wave w computes row blocks wr, wr+RW,
// ... (wr = w/2) against the CG/2 column groups starting at wc*CG/2 (wc = w%2).
template <bool GATEUP, int MB, int CG, int KH, int W>
__device__ __forceinline__ void gemm_tile(const GemmArgs &a, const TileInfo &ti, int nt0, int ntiles, int erot,
                                          uint8_t *smem) {
  static_assert(KH == 2, "8-row DMA units span a 64-wide K stage");
  using P = Pipe<MB, CG, KH, W>;
  constexpr int RW = W / 2;    // waves along the rows
  constexpr int NAM = P::NA_MAX, NB = P::NB, SA = P::SA, SB = P::SB, BK = P::BK;
  constexpr int MW = MB / RW;  // row blocks per wave
  constexpr int CW = CG / 2;   // column groups per wave
  constexpr int BN = GATEUP ? 16 * CG : 32 * CG;  // tile width (features or output columns)
  static_assert(W % 2 == 0, "waves form an RW x 2 grid");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int wr = wave >> 1, wc = wave & 1;
  const int K = GATEUP ? a.d : a.m;
  // routed tile: the routed experts' operands; appended dense-expert tile: its own
  const bf16_t *act = static_cast<const bf16_t *>(ti.sh ? a.sh_act : a.act);
  const int32_t *perm = ti.sh ? nullptr : a.perm;
  const void *w0 = ti.sh ? a.sh_w0 : a.w0;
  const void *w1 = ti.sh ? a.sh_w1 : a.w1;
  void *outp = ti.sh ? a.sh_out : a.out;
  // A units this wave stages per stage (wave-uniform): only units holding a row of
  // the tile (unit u covers rows 8u .. 8u+7); the MFMAs below skip row blocks past
  // the tile too, and rows past the tile are never stored
  const int fav = min(P::FA, (ti.rows + 7) >> 3);
  const int na = fav > wave ? (fav - wave + W - 1) / W : 0;
  const int ur = lane >> 3;  // DMA lane -> row in its unit

  // A units this wave stages: u = wave + W j -> row block u / 2, row half u % 2 (=
  // wave % 2).  Their token rows come through perm (routed tiles).  The perm loads
  // are issued from inline assembly ahead of the weight prologue and waited for
  // explicitly after it: a compiler-placed wait for them would be a vmcnt(0),
  // which also waits for the weight DMAs issued in between and so holds the
  // activation prologue back by a whole memory round trip.
  int srow[NAM];
#pragma unroll
  for (int j = 0; j < NAM; ++j) {
    const int u = min(wave + W * j, P::FA - 1);
    const int row = min((u >> 1) * 16 + (u & 1) * 8 + ur, ti.rows - 1);  // rows past the tile repeat its last row
    srow[j] = perm ? gload_i32(perm + ti.row0 + row) : ti.row0 + row;
  }
  // B units this wave stages: b = wave * NB + t -> block b / 2, row half t % 2
  const bf16_t *bsrc[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    const int b = wave * NB + t;
    const int blk = b >> 1, j = b & 1;
    const int fg = blk >> 1, cb = blk & 1;
    const int c = 8 * unit_chunk(lane);
    if (GATEUP) {
      const size_t f = static_cast<size_t>(ti.e) * a.m + nt0 * BN + fg * 16 + 8 * j + ur;
      bsrc[t] = static_cast<const bf16_t *>(cb ? w1 : w0) + f * a.d + c;
    } else {
      const size_t n = static_cast<size_t>(ti.e) * a.d + nt0 * BN + fg * 32 + cb * 16 + 8 * j + ur;
      bsrc[t] = static_cast<const bf16_t *>(w0) + n * a.m + c;
    }
  }
  // fragment read offsets inside a 16-row block (two units) for k halves 0 and 1
  const int rd_off0 = unit_read_offset(lane, 0), rd_off1 = unit_read_offset(lane, 1);
  const uint32_t ldsA = lds_addr(smem);
  const uint32_t ldsB = ldsA + SA * P::ASZ;
  const uint8_t *smemA = smem;
  const uint8_t *smemB = smem + SA * P::ASZ;

  f32x4_t acc[MW][2 * CW];
#pragma unroll
  for (int i = 0; i < MW; ++i)
#pragma unroll
    for (int c = 0; c < 2 * CW; ++c) acc[i][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  auto store_tile = [&](f32x4_t (&ac)[MW][2 * CW], int nt) {
    store_tile_impl<GATEUP, MW, CW, RW, BN>(a, ti, outp, ac, nt, wr, wc, r16, g);
  };

  const int nk = K / BK;
  // ntiles (1 or 2) N tiles of the M tile, nt0 and nt0 + 1, run as one pipeline
  // of NK = ntiles * nk stages: stage s is K block s % nk of tile s / nk, so the
  // second tile's first stages are in flight while the first tile's last steps
  // and its output stores run (no second prologue ramp)
  const int NK = ntiles * nk;
  const size_t tile_step = static_cast<size_t>(BN) * K;  // weight elements from one N tile to the next
  // Pipeline stage s covers K block (s + k0) % nk, k0 set by the tile's expert.
  // Experts start at different K blocks: rows 4 KB apart (d = 2048 bf16) read at
  // one K offset by every workgroup at once concentrate on a few HBM channels and
  // stream ~20% slower.  Every tile of one expert keeps one K order: the N tiles
  // of an M tile share its activation rows in their XCD's L2, and the M tiles of a
  // large expert that run at the same time on one XCD share its weight rows
  // (starting each M tile at its own block left them out of step, and the
  // wider-pool gate/up fetched three times its weight bytes from beyond L2).
  const int k0 = erot % nk;
  auto kofs = [&](int s) {
    s = s < nk ? s : s - nk;
    return (s + k0 < nk ? s + k0 : s + k0 - nk) * BK;
  };
  // weight units of stage s into LDS stage base st: weights that no other M tile
  // reads stream with the non-temporal hint; weights shared by several M tiles
  // (large experts, the dense expert's tiles) stay cacheable for the other tiles
  auto issue_b = [&](uint32_t st, int s) {
    const size_t o = (s < nk ? 0 : tile_step) + kofs(s);
    if (ti.once) {
#pragma unroll
      for (int t = 0; t < NB; ++t) dma16_stream(bsrc[t] + o, st + (wave * NB + t) * kFragBytes);
    } else {
#pragma unroll
      for (int t = 0; t < NB; ++t) dma16(bsrc[t] + o, st + (wave * NB + t) * kFragBytes);
    }
  };
  // prologue: B stages 0..SB-2, then A stages 0..SA-2
  for (int s = 0; s < SB - 1 && s < NK; ++s) {
    const uint32_t st = ldsB + s * P::BSZ;
    issue_b(st, s);
  }
  if (perm) {
    // the perm loads, issued before these weight DMAs (a constant count unless K is
    // shorter than the weight prologue)
    if (NK >= SB - 1)
      wait_vmcnt((SB - 1) * NB);
    else
      wait_vmcnt(NK * NB);
#pragma unroll
    for (int j = 0; j < NAM; ++j) reg_ready(srow[j]);
  }
  const bf16_t *asrc[NAM];
#pragma unroll
  for (int j = 0; j < NAM; ++j) asrc[j] = act + static_cast<size_t>(srow[j]) * K + 8 * unit_chunk(lane);
  for (int s = 0; s < SA - 1 && s < NK; ++s) {
    const uint32_t st = ldsA + s * P::ASZ;
#pragma unroll
    for (int j = 0; j < NAM; ++j)
      if (j < na) dma16(asrc[j] + kofs(s), st + (wave + W * j) * kFragBytes);
  }

  using CF = Closed<P>;
  for (int kt = 0; kt < NK; ++kt) {
    if (CF::on && na > 0) {
      if (CF::nb_pending(kt, NK))
        wait_vmcnt(NB);
      else
        wait_vmcnt(0);
    } else {
      wait_vmcnt(pending_ok<P>(kt, NK, na));
    }
    barrier();  // stage kt landed for every wave; every wave is done with stage kt-1
    if (kt + SA - 1 < NK) {
      const int s = kt + SA - 1;
      const uint32_t st = ldsA + (s % SA) * P::ASZ;
#pragma unroll
      for (int j = 0; j < NAM; ++j)
        if (j < na) dma16(asrc[j] + kofs(s), st + (wave + W * j) * kFragBytes);
    }
    const uint8_t *sa = smemA + (kt % SA) * P::ASZ;
    const uint8_t *sb = smemB + (kt % SB) * P::BSZ;
#pragma unroll
    for (int h = 0; h < KH; ++h) {
      bf16x8_t bf[2 * CW];  // [fl * 2 + cb]: column group wc*CW + fl, block cb
#pragma unroll
      for (int c = 0; c < 2 * CW; ++c)
        bf[c] = *reinterpret_cast<const bf16x8_t *>(sb + (2 * (wc * CW + (c >> 1)) + (c & 1)) * 2 * kFragBytes +
                                                    (h ? rd_off1 : rd_off0));
      // every row block's fragment is read up front, with the weight fragments
      // (blocks past the tile read stale LDS and are not multiplied): a read
      // placed after the branch below made each row block's MFMAs wait a full
      // LDS round trip
      bf16x8_t av[MW];
#pragma unroll
      for (int i = 0; i < MW; ++i)
        av[i] = *reinterpret_cast<const bf16x8_t *>(sa + (wr + RW * i) * 2 * kFragBytes + (h ? rd_off1 : rd_off0));
      // an empty use here keeps the compiler from sinking each read into the
      // branch that multiplies it
#pragma unroll
      for (int i = 0; i < MW; ++i) asm volatile("" ::"v"(av[i]));
#pragma unroll
      for (int i = 0; i < MW; ++i) {
        if ((wr + RW * i) * 16 >= ti.rows) break;  // wave-uniform: row blocks past the tile
#pragma unroll
        for (int c = 0; c < 2 * CW; ++c)
          acc[i][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bf[c], acc[i][c], 0, 0, 0);
      }
      // the weight DMAs of stage kt + SB - 1 go out behind the first k half's
      // MFMAs, so their issue (the memory pipeline's back-pressure) overlaps the
      // matrix cores instead of delaying them; the issue order, and so every
      // vmcnt count, is unchanged (A of a step, then its B)
      if (h == 0 && kt + SB - 1 < NK) {
        const int s = kt + SB - 1;
        issue_b(ldsB + (s % SB) * P::BSZ, s);
      }
    }
    if (kt == nk - 1 && ntiles > 1) {
      store_tile(acc, nt0);
#pragma unroll
      for (int i = 0; i < MW; ++i)
#pragma unroll
        for (int c = 0; c < 2 * CW; ++c) acc[i][c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
  }
  store_tile(acc, nt0 + ntiles - 1);
}

// tile width in features (gate/up) or output columns (down) for CG column groups
template <bool GATEUP> constexpr int tile_width(int cg) { return GATEUP ? 16 * cg : 32 * cg; }

// TPW (1 or 2): N tiles per workgroup, consecutive tiles of one M tile in one
// pipeline (gemm_tile).
template <bool GATEUP, int CG, int W, int TPW>
__global__ __launch_bounds__(W * 64) void grouped_gemm_bf16_kernel(GemmArgs a) {
  static_assert(TPW == 1 || TPW == 2, "one or two N tiles per workgroup");
  const int nN = (GATEUP ? a.m : a.d) / tile_width<GATEUP>(CG);
  const int nP = (nN + TPW - 1) / TPW;
  int grp, np;
  map_block(blockIdx.x, nP, &grp, &np);
  const int nt0 = np * TPW, ntiles = min(TPW, nN - nt0);
  const TileInfo ti = tile_info(a, grp);
  if (!ti.valid) return;
  __shared__ __align__(16) uint8_t smem[kLdsBytes];
  const int blocks = (ti.rows + 15) >> 4;
  // K rotation key: the expert (the appended dense expert gets its own)
  const int erot = ti.sh ? 0x155 : ti.e;
  if (blocks <= 4)
    gemm_tile<GATEUP, 4, CG, stage_halves<CG>(), W>(a, ti, nt0, ntiles, erot, smem);
  else if (blocks <= 8)
    gemm_tile<GATEUP, 8, CG, stage_halves<CG>(), W>(a, ti, nt0, ntiles, erot, smem);
  else if (blocks <= 12)
    gemm_tile<GATEUP, 12, CG, stage_halves<CG>(), W>(a, ti, nt0, ntiles, erot, smem);
  else
    gemm_tile<GATEUP, 16, CG, stage_halves<CG>(), W>(a, ti, nt0, ntiles, erot, smem);
}

// ------------------------------------------------------------------ fp32 (MFMA)
// fp32 layers (the small parity workloads): v_mfma_f32_16x16x4f32 on fp32
// operands staged in LDS 16 k at a time.  A workgroup (4 waves) takes one M tile
// (up to 256 rows) and one N tile of 16 features (gate/up: a gate block and an
// up block) or 16 output columns (down); wave w multiplies row blocks w, w+4,
// w+8, w+12.  Operand lanes: A row l%16 / B column l%16, k = l/16 of the
// instruction's 4.
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
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r16 = lane & 15, g = lane >> 4;
  const int d = a.d, m = a.m, f0 = nt * F_BN;
  const int nrb = (ti.rows + 15) >> 4;
  const float *xn = static_cast<const float *>(a.act);
  const float *wg = static_cast<const float *>(a.w0);
  const float *wu = static_cast<const float *>(a.w1);
  f32x4_t accg[4], accu[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) accg[i] = accu[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < d; k0 += F_BK) {
    for (int c = tid; c < kTileM * F_BK; c += 256) {
      const int r = c >> 4, kk = c & 15;
      float v = 0.f;
      if (r < ti.rows) {
        const int tok = a.perm ? a.perm[ti.row0 + r] : ti.row0 + r;
        v = xn[static_cast<size_t>(tok) * d + k0 + kk];
      }
      As[r][kk] = v;
    }
    {
      const int r = tid >> 4, kk = tid & 15;
      const size_t wrow = (static_cast<size_t>(ti.e) * m + f0 + r) * d + k0 + kk;
      Bg[r][kk] = wg[wrow];
      Bu[r][kk] = wu[wrow];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < F_BK / 4; ++j) {
      const float bgv = Bg[r16][4 * j + g], buv = Bu[r16][4 * j + g];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rb = wave + 4 * i;
        if (rb >= nrb) break;  // wave-uniform
        const float av = As[rb * 16 + r16][4 * j + g];
        accg[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bgv, accg[i], 0, 0, 0);
        accu[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, buv, accu[i], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  // lane holds feature f0 + r16 of rows 16 rb + 4 g + q
  float *H = static_cast<float *>(a.out);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = (wave + 4 * i) * 16 + 4 * g + q;
      if (r < ti.rows) H[static_cast<size_t>(ti.row0 + r) * m + f0 + r16] = silu(accg[i][q]) * accu[i][q];
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
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r16 = lane & 15, g = lane >> 4;
  const int d = a.d, m = a.m, n0 = nt * F_BN;
  const int nrb = (ti.rows + 15) >> 4;
  const float *H = static_cast<const float *>(a.act);
  const float *wd = static_cast<const float *>(a.w0);
  f32x4_t acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < m; k0 += F_BK) {
    for (int c = tid; c < kTileM * F_BK; c += 256) {
      const int r = c >> 4, kk = c & 15;
      As[r][kk] = (r < ti.rows) ? H[static_cast<size_t>(ti.row0 + r) * m + k0 + kk] : 0.f;
    }
    {
      const int r = tid >> 4, kk = tid & 15;
      Bs[r][kk] = wd[(static_cast<size_t>(ti.e) * d + n0 + r) * m + k0 + kk];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < F_BK / 4; ++j) {
      const float bv = Bs[r16][4 * j + g];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rb = wave + 4 * i;
        if (rb >= nrb) break;  // wave-uniform
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(As[rb * 16 + r16][4 * j + g], bv, acc[i], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  float *Y = static_cast<float *>(a.out);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = (wave + 4 * i) * 16 + 4 * g + q;
      if (r < ti.rows) Y[static_cast<size_t>(ti.row0 + r) * d + n0 + r16] = acc[i][q];
    }
}

// N tiles per workgroup.  Down: two (K is only m deep, so a tile is a short
// pipeline; the pair runs as one and the grid is one round of workgroups fewer:
// wider-pool down 153.9 -> 149.3 us, the 4096-token layer's unchanged).  Gate/up:
// one.  Two, three or four made it 9-50% slower, three even where its grid is
// exactly one round on the 256 CUs: with one tile per workgroup the N tiles of an
// M tile run at once on one XCD and share the gathered activation rows in its L2,
// while a workgroup walking its tiles one after the other gathers them again for
// each tile.
constexpr int kTpwGateUp = 1;
constexpr int kTpwDown = 2;
int pairs(int nN, int tpw) { return (nN + tpw - 1) / tpw; }

unsigned grid_for(int max_groups, int nN) {
  const int g8 = (max_groups + 7) / 8;
  return static_cast<unsigned>(8 * nN * g8);
}

}  // namespace

hipError_t launch_gateup(const GemmArgs &a, bool bf16, hipStream_t stream) {
  if (a.max_groups <= 0) return hipSuccess;
  if (bf16)
  {
    // 128 features per tile when they divide m, else 64
    if (a.m % tile_width<true>(8) == 0)
      grouped_gemm_bf16_kernel<true, 8, kGemmWaves, kTpwGateUp>
          <<<dim3(grid_for(a.max_groups, pairs(a.m / tile_width<true>(8), kTpwGateUp))), kGemmWaves * 64, 0,
             stream>>>(a);
    else
      grouped_gemm_bf16_kernel<true, 4, kGemmWaves, kTpwGateUp>
          <<<dim3(grid_for(a.max_groups, pairs(a.m / tile_width<true>(4), kTpwGateUp))), kGemmWaves * 64, 0,
             stream>>>(a);
  }
  else
    gateup_f32_kernel<<<dim3(grid_for(a.max_groups, a.m / F_BN)), 256, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_down(const GemmArgs &a, bool bf16, hipStream_t stream) {
  if (a.max_groups <= 0) return hipSuccess;
  if (bf16)
  {
    // 256 output columns per tile when they divide d, else 128
    if (a.d % tile_width<false>(8) == 0)
      grouped_gemm_bf16_kernel<false, 8, kGemmWaves, kTpwDown>
          <<<dim3(grid_for(a.max_groups, pairs(a.d / tile_width<false>(8), kTpwDown))), kGemmWaves * 64, 0,
             stream>>>(a);
    else
      grouped_gemm_bf16_kernel<false, 4, kGemmWaves, kTpwDown>
          <<<dim3(grid_for(a.max_groups, pairs(a.d / tile_width<false>(4), kTpwDown))), kGemmWaves * 64, 0,
             stream>>>(a);
  }
  else
    down_f32_kernel<<<dim3(grid_for(a.max_groups, a.d / F_BN)), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
