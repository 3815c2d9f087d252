// Dispatch plan: expert histogram, exclusive prefix sum and the compacted
// permutation of kept slots, plus the M-tile list the grouped GEMMs walk.
//
// The layer evaluates only the experts indexed by each token's active set
// (Alg. 1's online loop).  The router kernel leaves one bit per kept
// (expert, token) pair in a per-expert token bitmap; here one workgroup of 1024
// threads turns the bitmap into
//   counts[e]   = popcount of expert e's bitmap,
//   offsets[e]  = exclusive prefix sum of counts,
//   perm[r]     = token of compacted row r, rows ordered by (expert, token),
//   slot_row    = compacted row of every kept (token, slot),
//   tiles       = (expert, first row, rows) of every kTileM-row M tile.
// The order is fixed by the bitmap, so the plan is bit-exact and independent
// of how the router workgroups were scheduled.  P = 1024 / N threads share an
// expert, each owning a contiguous run of bitmap words: pass 1 counts, a
// wavefront scan over experts places them, pass 2 writes rows in token order.
#include "ace_internal.h"

namespace ace {

namespace {

__device__ __forceinline__ int wave_inclusive_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int n = __shfl_up(v, off);
    if (lane >= off) v += n;
  }
  return v;
}

__global__ __launch_bounds__(1024) void plan_kernel(PlanArgs a) {
  __shared__ int cnt[1024];
  __shared__ int ecount[kMaxN];
  __shared__ int eoff[kMaxN + 1];
  __shared__ int tcount[kMaxN];
  __shared__ int toff[kMaxN + 1];

  const int tid = threadIdx.x;
  const int N = a.N;
  const int W = a.W;
  const int P = 1024 / N;
  const int e = tid / P;
  const int p = tid - e * P;
  const bool active = e < N;
  const int cw = (W + P - 1) / P;
  const int w0 = active ? min(W, p * cw) : 0;
  const int w1 = active ? min(W, w0 + cw) : 0;
  const unsigned long long *bm = a.bitmap + static_cast<size_t>(active ? e : 0) * W;

  int c = 0;
  for (int w = w0; w < w1; ++w) c += __popcll(bm[w]);
  cnt[tid] = c;
  __syncthreads();

  if (tid < N) {
    int s = 0;
    for (int q = 0; q < P; ++q) s += cnt[tid * P + q];
    ecount[tid] = s;
    tcount[tid] = (s + kTileM - 1) / kTileM;
  }
  __syncthreads();

  if (tid < 64) {
    // each lane scans 4 consecutive experts (N <= 256)
    int loc[4], tloc[4];
    int s = 0, ts = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int ee = tid * 4 + j;
      loc[j] = s;
      tloc[j] = ts;
      s += (ee < N) ? ecount[ee] : 0;
      ts += (ee < N) ? tcount[ee] : 0;
    }
    const int incl = wave_inclusive_scan(s, tid);
    const int tincl = wave_inclusive_scan(ts, tid);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int ee = tid * 4 + j;
      if (ee < N) {
        eoff[ee] = incl - s + loc[j];
        toff[ee] = tincl - ts + tloc[j];
      }
    }
    if (tid == 63) {
      eoff[N] = incl;
      toff[N] = tincl;
    }
  }
  __syncthreads();

  if (tid < N) {
    a.counts[tid] = ecount[tid];
    a.offsets[tid] = eoff[tid];
    const int nt = tcount[tid];
    for (int j = 0; j < nt; ++j) {
      const int g = toff[tid] + j;
      a.tile_expert[g] = tid;
      a.tile_row0[g] = eoff[tid] + j * kTileM;
      a.tile_rows[g] = min(kTileM, ecount[tid] - j * kTileM);
    }
  }
  if (tid == 0) {
    a.offsets[N] = eoff[N];
    a.n_tiles[0] = toff[N];
  }

  if (active) {
    int row = eoff[e];
    for (int q = 0; q < p; ++q) row += cnt[e * P + q];
    for (int w = w0; w < w1; ++w) {
      unsigned long long bits = bm[w];
      while (bits) {
        const int b = __builtin_ctzll(bits);
        bits &= bits - 1ull;
        const int t = w * 64 + b;
        a.perm[row] = t;
        const int32_t *ids = a.topk_idx + static_cast<size_t>(t) * a.k;
        for (int i = 0; i < a.k; ++i)
          if (ids[i] == e) a.slot_row[static_cast<size_t>(t) * a.k + i] = row;
        ++row;
      }
    }
  }
}

}  // namespace

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
  plan_kernel<<<dim3(1), 1024, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
