// Pipeline geometry and exact vmcnt waits of the grouped expert GEMMs (shared by
// the kernels and by the host-side check that replays every issue sequence).
//
// A tile of MB 16-row blocks (MB a multiple of 4), CG column groups (gate/up: 16
// features each, a gate and an up block; down: 32 output columns, two blocks) and
// KH 32-wide k halves per stage (BK = 32 KH) streams its operands through two LDS
// rings: A (activation rows, mostly L2 hits) and B (expert weights, from HBM).  A
// stage of A holds MB*KH units spread over the W waves (a wave stages na <=
// NA_MAX of them); a stage of B holds 2*CG*KH units, NB per wave.  One unit is
// one DMA instruction (1 KB).
#pragma once

#include <hip/hip_runtime.h>

namespace ace {

constexpr int kPipeUnitBytes = 1024;       // one DMA unit
constexpr int kPipeLdsBytes = 160 * 1024;  // LDS of one workgroup

__host__ __device__ constexpr int pipe_min(int a, int b) { return a < b ? a : b; }
__host__ __device__ constexpr int pipe_max(int a, int b) { return a > b ? a : b; }

template <int MB, int CG, int KH, int W> struct Pipe {
  static constexpr int BK = 32 * KH;
  static constexpr int FA = MB * KH;                      // A units per stage
  static constexpr int NA_MAX = (FA + W - 1) / W;
  static constexpr int NB = 2 * CG * KH / W;              // B DMAs per wave per stage
  static constexpr int ASZ = FA * kPipeUnitBytes;
  static constexpr int BSZ = 2 * CG * KH * kPipeUnitBytes;
  static constexpr int SA = KH == 2 ? ((MB >= 16 || (CG >= 8 && MB >= 8)) ? 2 : MB >= 8 ? 3 : 4) : 4;
  static constexpr int SB0 = (kPipeLdsBytes - SA * ASZ) / BSZ;
  static constexpr int SBMAX = KH == 2 ? 8 : 10;
  static constexpr int SB = SB0 > SBMAX ? SBMAX : SB0;
  static_assert(2 * CG * KH % W == 0, "B units must spread evenly over the waves");
  static_assert(SB >= 2 && SA >= 2, "ring too shallow");
  static_assert(SA * ASZ + SB * BSZ <= kPipeLdsBytes, "rings exceed LDS");
  static_assert((SA - 1) * NA_MAX + (SB - 1) * NB + NA_MAX + NB <= 63, "outstanding DMAs exceed the wait table");
};

// A wave's DMA issue sequence: a prologue of B stages 0..PB-1 then A stages
// 0..PA-1 (PB = min(SB-1, nk), PA = min(SA-1, nk)); then iteration j issues
// A(j+SA-1) and then B(j+SB-1), each only if it exists.  cum_ops(j) = DMAs
// issued before iteration j.
template <class P>
__host__ __device__ inline int cum_ops(int j, int nk, int na) {
  const int PB = pipe_min(P::SB - 1, nk), PA = pipe_min(P::SA - 1, nk);
  return PB * P::NB + PA * na + pipe_max(0, pipe_min(j, nk - P::SA + 1)) * na +
         pipe_max(0, pipe_min(j, nk - P::SB + 1)) * P::NB;
}

// DMAs that may still be outstanding at the wait before stage kt's compute:
// everything issued after the later of A(kt) and B(kt) (vmcnt completes in
// issue order).  na = this wave's A DMAs per stage.
template <class P>
__host__ __device__ inline int pending_ok(int kt, int nk, int na) {
  const int PB = pipe_min(P::SB - 1, nk), PA = pipe_min(P::SA - 1, nk);
  int end_a, end_b;
  if (na == 0) {
    end_a = 0;  // this wave stages no A units
  } else if (kt < PA) {
    end_a = PB * P::NB + (kt + 1) * na;
  } else {
    end_a = cum_ops<P>(kt - P::SA + 1, nk, na) + na;
  }
  if (kt < PB) {
    end_b = (kt + 1) * P::NB;
  } else {
    const int i = kt - P::SB + 1;
    end_b = cum_ops<P>(i, nk, na) + (i + P::SA - 1 < nk ? na : 0) + P::NB;
  }
  return cum_ops<P>(kt, nk, na) - pipe_max(end_a, end_b);
}

// Closed form for SA == 2 < SB.  A wave that stages A units (na > 0) issues A(0)
// last in its prologue and A(kt) as the first DMA of iteration kt - 1, followed in
// that iteration only by B(kt + SB - 2) when that stage exists; B(kt) always went
// out earlier.  So the wait before stage kt allows NB DMAs when kt >= 1 and
// kt + SB - 2 < nk, and none otherwise: two constant waits, which spare the
// run-time count and its branch tree in every step.
template <class P> struct Closed {
  static constexpr bool on = P::SA == 2 && P::SB > 2;
  __host__ __device__ static bool nb_pending(int kt, int nk) { return kt >= 1 && kt + P::SB - 2 < nk; }
};

}  // namespace ace
