// Dispatch plan: expert histogram, exclusive prefix sum and the compacted
// permutation of kept slots, plus the M-tile list the grouped GEMMs walk.
//
// The layer evaluates only the experts indexed by each token's active set
// (Alg. 1's online loop).  Compacted rows are ordered by (expert, token).  The
// router kernel leaves, per 16-token chunk g and expert e, the kept count
// chunk_count[g][e] and, per kept slot, its rank among the chunk's kept slots
// of that expert.  Two kernels finish the plan:
//   expert_scan (one workgroup per expert): chunk_base[e][g] = sum of
//     chunk_count[g'][e] over g' < g, and counts[e];
//   scatter (one workgroup per chunk): offsets = exclusive prefix sum of counts
//     (each workgroup recomputes it; N <= 256), then every kept slot writes
//     row = offsets[e] + chunk_base[e][g] + local_rank into perm and slot_row.
//     Workgroup 0 also writes offsets and the M-tile list.
// Integer work only, no atomics: the plan is bit-exact and independent of
// scheduling.
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

// exclusive scan of v[0..n) (n <= 256) by one wavefront into out[0..n]
__device__ __forceinline__ void wave_scan_256(const int *v, int *out, int n, int lane) {
  int loc[4];
  int s = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = lane * 4 + j;
    loc[j] = s;
    s += (i < n) ? v[i] : 0;
  }
  const int incl = wave_inclusive_scan(s, lane);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = lane * 4 + j;
    if (i < n) out[i] = incl - s + loc[j];
  }
  if (lane == 63) out[n] = incl;
}

__global__ __launch_bounds__(256) void expert_scan_kernel(PlanArgs a) {
  __shared__ int part[256];
  const int e = blockIdx.x;
  const int tid = threadIdx.x;
  const int G = a.G, N = a.N;
  const int per = (G + 255) / 256;
  const int g0 = min(G, tid * per), g1 = min(G, g0 + per);
  int s = 0;
  for (int g = g0; g < g1; ++g) s += a.chunk_count[static_cast<size_t>(g) * N + e];
  part[tid] = s;
  __syncthreads();
  if (tid < 64) {
    // exclusive scan of the 256 partial sums
    int loc[4];
    int acc = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      loc[j] = acc;
      acc += part[tid * 4 + j];
    }
    const int incl = wave_inclusive_scan(acc, tid);
#pragma unroll
    for (int j = 0; j < 4; ++j) part[tid * 4 + j] = incl - acc + loc[j];
    if (tid == 63) a.counts[e] = incl;
  }
  __syncthreads();
  int run = part[tid];
  int32_t *base = a.chunk_base + static_cast<size_t>(e) * G;
  for (int g = g0; g < g1; ++g) {
    base[g] = run;
    run += a.chunk_count[static_cast<size_t>(g) * N + e];
  }
}

__global__ __launch_bounds__(128) void scatter_kernel(PlanArgs a) {
  __shared__ int cnt[kMaxN];
  __shared__ int off[kMaxN + 1];
  __shared__ int tcnt[kMaxN];
  __shared__ int toff[kMaxN + 1];
  const int tid = threadIdx.x;
  const int N = a.N;
  const int g = blockIdx.x;
  for (int e = tid; e < N; e += 128) {
    cnt[e] = a.counts[e];
    tcnt[e] = (cnt[e] + kTileM - 1) / kTileM;
  }
  __syncthreads();
  if (tid < 64) {
    wave_scan_256(cnt, off, N, tid);
    if (g == 0) wave_scan_256(tcnt, toff, N, tid);
  }
  __syncthreads();

  if (g == 0) {
    for (int e = tid; e <= N; e += 128) a.offsets[e] = off[e];
    if (tid == 0) a.n_tiles[0] = toff[N];
    for (int e = tid; e < N; e += 128) {
      for (int j = 0; j < tcnt[e]; ++j) {
        const int tg = toff[e] + j;
        a.tile_expert[tg] = e;
        a.tile_row0[tg] = off[e] + j * kTileM;
        a.tile_rows[tg] = min(kTileM, cnt[e] - j * kTileM);
      }
    }
  }

  const int k = a.k;
  if (tid < kRouteTokens * k) {
    const int tl = tid / k;
    const int t = g * kRouteTokens + tl;
    if (t < a.T) {
      const size_t o = static_cast<size_t>(t) * k + (tid - tl * k);
      if (a.keep[o]) {
        const int e = a.topk_idx[o];
        const int row = off[e] + a.chunk_base[static_cast<size_t>(e) * a.G + g] + a.local_rank[o];
        a.perm[row] = t;
        a.slot_row[o] = row;
      }
    }
  }
}

}  // namespace

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
  expert_scan_kernel<<<dim3(a.N), 256, 0, stream>>>(a);
  scatter_kernel<<<dim3(a.G), 128, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
