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
// When the [G, N] count matrix is at most 128 KB (and N a multiple of 4),
// plan_kernel does both in one launch: each chunk workgroup reads the matrix and
// derives the totals and its own chunk base itself.  Integer work only, no atomics: the plan is bit-exact
// and independent of scheduling.
#include <type_traits>

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

constexpr int kPlanMaxBytes = 128 * 1024;  // count matrix size up to which one kernel plans
#ifndef ACE_PLAN_LPT
#define ACE_PLAN_LPT 1
#endif

// One kernel for the whole plan when the [G, N] count matrix is small: every
// chunk workgroup reads the whole matrix (L2-resident after the first reads) and
// derives each expert's total and its own chunk base (the part of the column
// before chunk g) itself, then scatters its kept slots.  Workgroup 0 also writes
// counts, offsets and the M-tile list.  The same integers as expert_scan +
// scatter, in one launch.
//
// Column sums: thread (r, w) reads V 32-bit words (4V experts) of chunk rows
// r, r + R, ... and adds their bytes as packed 16-bit lanes (even bytes, odd
// bytes); a chunk holds at most 16 tokens, so a lane stays below 16 * ceil(G / R)
// (checked on the host).  The R row groups are then added per expert.
template <int V>
__global__ __launch_bounds__(256) void plan_kernel(PlanArgs a) {
  __shared__ uint32_t red[4][256 * V];  // even/odd byte sums, then the same before chunk g
  __shared__ int base[kMaxN];
  __shared__ int cnt[kMaxN], off[kMaxN + 1], tcnt[kMaxN], toff[kMaxN + 1];
  typedef typename std::conditional<V == 4, uint4, uint32_t>::type word_t;
  const int tid = threadIdx.x;
  const int N = a.N, G = a.G, g = blockIdx.x;
  const int NW = N / 4;        // words per chunk row
  const int W = NW / V;        // threads per chunk row
  const int R = 256 / W;       // row groups
  const int r = tid / W, w = tid - r * W;
  // this thread's slot of the chunk (thread tid < 16 k): its routing, loaded
  // now so the loads overlap the column sums below
  const int k = a.k;
  const int tl = tid / k;
  const int t = g * kRouteTokens + tl;
  const bool has_slot = tid < kRouteTokens * k && t < a.T;
  const size_t o = static_cast<size_t>(t) * k + (tid - tl * k);
  const bool kept = has_slot && a.keep[o];
  const int e_slot = has_slot ? a.topk_idx[o] : 0;
  const int rank = has_slot ? a.local_rank[o] : 0;
  if (r < R) {
    uint32_t ev[V], od[V], pev[V], pod[V];
#pragma unroll
    for (int j = 0; j < V; ++j) ev[j] = od[j] = pev[j] = pod[j] = 0;
    const word_t *src = reinterpret_cast<const word_t *>(a.chunk_count) + w;
    for (int c0 = r; c0 < G; c0 += 8 * R) {
      word_t q[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = c0 + u * R;
        if (c < G) q[u] = src[static_cast<size_t>(c) * W];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = c0 + u * R;
        if (c >= G) break;
        const uint32_t before = c < g ? 0xffffffffu : 0u;
        const uint32_t *qw = reinterpret_cast<const uint32_t *>(&q[u]);
#pragma unroll
        for (int j = 0; j < V; ++j) {
          const uint32_t e0 = qw[j] & 0x00ff00ffu, o0 = (qw[j] >> 8) & 0x00ff00ffu;
          ev[j] += e0;
          od[j] += o0;
          pev[j] += e0 & before;
          pod[j] += o0 & before;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int i = r * NW + w * V + j;
      red[0][i] = ev[j];
      red[1][i] = od[j];
      red[2][i] = pev[j];
      red[3][i] = pod[j];
    }
  }
  __syncthreads();
  if (tid < N) {
    const int wi = tid >> 2, b = tid & 3;
    const int q = b & 1, sh = 16 * (b >> 1);
    int t = 0, p = 0;
    for (int rr = 0; rr < R; ++rr) {
      t += (red[q][rr * NW + wi] >> sh) & 0xffffu;
      p += (red[q + 2][rr * NW + wi] >> sh) & 0xffffu;
    }
    cnt[tid] = t;
    tcnt[tid] = (t + kTileM - 1) / kTileM;
    base[tid] = p;
  }
  __syncthreads();
  if (tid < 64) {
    wave_scan_256(cnt, off, N, tid);
    if (g == 0) wave_scan_256(tcnt, toff, N, tid);
  }
  __syncthreads();
  if (g == 0) {
    for (int e = tid; e < N; e += 256) {
      a.counts[e] = cnt[e];
      for (int j = 0; j < tcnt[e]; ++j) {
        const int tg = toff[e] + j;
        a.tile_expert[tg] = e;
        a.tile_row0[tg] = off[e] + j * kTileM;
        a.tile_rows[tg] = min(kTileM, cnt[e] - j * kTileM);
      }
    }
    for (int e = tid; e <= N; e += 256) a.offsets[e] = off[e];
    if (tid == 0) a.n_tiles[0] = toff[N];
  }
  // The gate/up launch's tile order.  When every expert fits one M tile, longest
  // first (rows descending, then expert id): its grid takes tiles in this order,
  // so the longest tiles start first and the last round of workgroups holds the
  // short ones.  Otherwise list order, which keeps an expert's tiles adjacent
  // (their grid neighbours share its weights in L2).  The down launch keeps list
  // order: there, concurrent workgroups then read and write neighbouring H and Y
  // rows (longest first measured slower for it).  Workgroup g places experts g,
  // g + G, ...: the position is the count of experts with more rows, or as many
  // rows and a lower id (one block-wide count per expert); its list index is the
  // count of active experts with a lower id.
  if (a.tile_order) {
    if (ACE_PLAN_LPT && !__syncthreads_or(tid < N && tcnt[tid] > 1)) {
      for (int e = g; e < N; e += G) {
        const int ce = cnt[e];
        const int pos = __syncthreads_count(tid < N && (cnt[tid] > ce || (cnt[tid] == ce && tid < e)));
        const int idx = __syncthreads_count(tid < e && cnt[tid] > 0);
        if (tid == 0 && ce > 0) a.tile_order[pos] = idx;
      }
    } else if (g == 0) {
      for (int i = tid; i < toff[N]; i += 256) a.tile_order[i] = i;
    }
  }
  // this chunk's kept slots: row = offsets[e] + chunk base of e + rank in the chunk
  if (kept) {
    const int row = off[e_slot] + base[e_slot] + rank;
    a.perm[row] = t;
    a.slot_row[o] = row;
  }
}

}  // namespace

// one-kernel plan: small matrix, rows of whole words, 16-bit lane sums that cannot overflow
static bool plan_one_kernel(const PlanArgs &a) {
  const long long bytes = static_cast<long long>(a.G) * a.N;
  const int V = a.N % 16 == 0 ? 4 : 1;
  const int R = a.N % 4 == 0 ? 256 / (a.N / 4 / V) : 0;
  return bytes <= kPlanMaxBytes && R > 0 && 16LL * ((a.G + R - 1) / R) <= 0xffff;
}

bool plan_writes_order(const PlanArgs &a) { return plan_one_kernel(a); }

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
  const int V = a.N % 16 == 0 ? 4 : 1;
  if (plan_one_kernel(a)) {
    if (V == 4)
      plan_kernel<4><<<dim3(a.G), 256, 0, stream>>>(a);
    else
      plan_kernel<1><<<dim3(a.G), 256, 0, stream>>>(a);
  } else {
    expert_scan_kernel<<<dim3(a.N), 256, 0, stream>>>(a);
    scatter_kernel<<<dim3(a.G), 128, 0, stream>>>(a);
  }
  return hipGetLastError();
}

}  // namespace ace
