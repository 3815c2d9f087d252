// Budget-to-threshold mapping (App. C.1) on the device: from the contribution
// scores c [n_rows, k] of one score pass (one or more layers), the threshold
// tau_q for each requested skip ratio q.
//
//  * N_all = n_rows * k routed slots.  Candidates exclude slot 0 (the top-1
//    expert) and, with m_min > 1, the m_min - 1 highest-c other slots of each
//    row (ties to the lower slot): Alg. 4's restore step never skips them.
//  * m_q = clip(round-half-even(q N_all), 0, N_cand); tau_q lies between the
//    m_q-th and (m_q+1)-th smallest candidate scores: their midpoint when they
//    differ; at a tie on value v, tau = v (realising #{c < v}) or the midpoint
//    of v and the next larger score (realising #{c <= v}), whichever count is
//    closer to m_q, the lower one on a draw; m_q = 0 gives 0, m_q = N_cand +inf.
//  * The order statistics come from a radix select on 32-bit order-preserving
//    keys: four 8-bit digit passes, each a histogram of the candidates that
//    still match the digits chosen so far (LDS histograms, integer atomics into
//    global memory) followed by a one-block pick of the digit holding the rank.
//    All counting is integer, so the result is exact and deterministic; the
//    midpoint is formed in fp64 from the two fp32 scores and rounded once.
// Every step runs on the caller's stream with no host synchronisation; ranks
// that depend on earlier results are read from device memory.
#include "ace_internal.h"

namespace ace {

namespace {

constexpr int kJobs = 2 * kTauMaxQ;  // two order statistics per budget
constexpr int kBins = 256;

struct Job {
  unsigned long long rank;  // remaining rank inside the current prefix (0-based)
  uint32_t prefix;          // key digits fixed so far
  int active;
};

struct TauState {
  unsigned long long n_cand;
  long long m_q[kTauMaxQ];
  unsigned long long below[kTauMaxQ], above[kTauMaxQ];  // #{c < v}, #{c <= v} at a boundary tie
  uint32_t lo[kTauMaxQ], hi[kTauMaxQ], next[kTauMaxQ];  // keys of c_(m_q), c_(m_q+1), next above v
  int mode[kTauMaxQ];  // 0: zero / inf / midpoint decided by lo, hi; 1: tie, tau = v; 2: tie, midpoint to next; 3: tie, inf
  Job job[kJobs];
};

struct TauArgs {
  const float *scores;
  long long n_rows;
  int k, m_min, n_q;
  double q[kTauMaxQ];
  TauState *st;
  unsigned long long *hist;  // [kJobs][kBins]
  float *tau;
  long long *m_q_out;        // optional
  long long *n_cand_out;     // optional
};

// order-preserving key of a non-NaN float (-0 taken as +0)
__device__ __forceinline__ uint32_t key_of(float c) {
  const uint32_t u = __float_as_uint(c + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float value_of(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// candidate slots of one row: bit i set if slot i may be skipped
__device__ __forceinline__ unsigned row_candidates(const float (&c)[kMaxK], int k, int m_min) {
  unsigned cand = 0;
#pragma unroll
  for (int i = 1; i < kMaxK; ++i) {
    int rank = 0;  // higher-c other slots (ties: lower slot first)
#pragma unroll
    for (int j = 1; j < kMaxK; ++j)
      if (j < k && j != i && (c[j] > c[i] || (c[j] == c[i] && j < i))) ++rank;
    if (i < k && rank >= m_min - 1) cand |= 1u << i;
  }
  return cand;
}

__device__ __forceinline__ void load_row(const TauArgs &a, long long r, float (&c)[kMaxK]) {
#pragma unroll
  for (int i = 0; i < kMaxK; ++i) c[i] = i < a.k ? a.scores[r * a.k + i] : 0.f;
}

__global__ __launch_bounds__(256) void tau_init_kernel(TauArgs a) {
  const int tid = threadIdx.x;
  for (int i = tid; i < kJobs * kBins; i += 256) a.hist[i] = 0ull;
  if (tid == 0) {
    TauState &s = *a.st;
    s.n_cand = 0;
    for (int i = 0; i < kTauMaxQ; ++i) {
      s.m_q[i] = 0;
      s.below[i] = s.above[i] = 0;
      s.lo[i] = s.hi[i] = s.next[i] = 0;
      s.mode[i] = 0;
    }
    for (int j = 0; j < kJobs; ++j) s.job[j] = Job{0ull, 0u, 0};
  }
}

__device__ __forceinline__ unsigned long long block_sum(unsigned long long v) {
  __shared__ unsigned long long part[4];
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  const unsigned long long t = part[0] + part[1] + part[2] + part[3];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(256) void tau_count_kernel(TauArgs a) {
  unsigned long long n = 0;
  for (long long r = blockIdx.x * 256ll + threadIdx.x; r < a.n_rows; r += 256ll * gridDim.x) {
    float c[kMaxK];
    load_row(a, r, c);
    n += __popc(row_candidates(c, a.k, a.m_min));
  }
  n = block_sum(n);
  if (threadIdx.x == 0 && n) atomicAdd(&a.st->n_cand, n);
}

__global__ void tau_setup_kernel(TauArgs a) {
  if (threadIdx.x != 0) return;
  TauState &s = *a.st;
  const double n_all = static_cast<double>(a.n_rows) * a.k;
  const long long nc = static_cast<long long>(s.n_cand);
  for (int i = 0; i < a.n_q; ++i) {
    long long m = static_cast<long long>(rint(a.q[i] * n_all));
    m = m < 0 ? 0 : (m > nc ? nc : m);
    s.m_q[i] = m;
    const bool inner = m > 0 && m < nc;
    s.job[2 * i] = Job{static_cast<unsigned long long>(inner ? m - 1 : 0), 0u, inner ? 1 : 0};
    s.job[2 * i + 1] = Job{static_cast<unsigned long long>(inner ? m : 0), 0u, inner ? 1 : 0};
  }
}

// histogram of digit `pass` (0 = most significant) of the candidates matching each active job's prefix
__global__ __launch_bounds__(256) void tau_hist_kernel(TauArgs a, int pass) {
  __shared__ uint32_t h[kJobs][kBins];
  __shared__ uint32_t pref[kJobs];
  __shared__ int act[kJobs];
  for (int i = threadIdx.x; i < kJobs * kBins; i += 256) (&h[0][0])[i] = 0u;
  if (threadIdx.x < kJobs) {
    pref[threadIdx.x] = a.st->job[threadIdx.x].prefix;
    act[threadIdx.x] = a.st->job[threadIdx.x].active;
  }
  __syncthreads();
  const int shift = 24 - 8 * pass;
  const uint32_t mask = pass == 0 ? 0u : (0xFFFFFFFFu << (32 - 8 * pass));
  for (long long r = blockIdx.x * 256ll + threadIdx.x; r < a.n_rows; r += 256ll * gridDim.x) {
    float c[kMaxK];
    load_row(a, r, c);
    const unsigned cand = row_candidates(c, a.k, a.m_min);
#pragma unroll
    for (int i = 1; i < kMaxK; ++i) {
      if (!((cand >> i) & 1u)) continue;
      const uint32_t key = key_of(c[i]);
      const uint32_t digit = (key >> shift) & 0xFFu;
      for (int j = 0; j < kJobs; ++j)
        if (act[j] && (key & mask) == pref[j]) atomicAdd(&h[j][digit], 1u);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kJobs * kBins; i += 256) {
    const uint32_t v = (&h[0][0])[i];
    if (v) atomicAdd(&a.hist[i], static_cast<unsigned long long>(v));
  }
}

// one block per job: the digit whose cumulative count passes the job's rank
__global__ __launch_bounds__(256) void tau_pick_kernel(TauArgs a, int pass) {
  const int j = blockIdx.x;
  Job &job = a.st->job[j];
  unsigned long long *hist = a.hist + static_cast<size_t>(j) * kBins;
  __shared__ unsigned long long cum[kBins];
  const int b = threadIdx.x;
  cum[b] = hist[b];
  __syncthreads();
  // inclusive scan over the 256 bins (Hillis-Steele)
  for (int off = 1; off < kBins; off <<= 1) {
    const unsigned long long v = b >= off ? cum[b - off] : 0ull;
    __syncthreads();
    cum[b] += v;
    __syncthreads();
  }
  const int active = job.active;
  const unsigned long long rank = job.rank;
  __syncthreads();
  if (active) {
    const unsigned long long before = b > 0 ? cum[b - 1] : 0ull;
    if (rank >= before && rank < cum[b]) {  // exactly one bin holds the rank
      job.rank = rank - before;
      job.prefix |= static_cast<uint32_t>(b) << (24 - 8 * pass);
    }
  }
  hist[b] = 0ull;  // ready for the next pass
}

// after the first select: record the keys; at a boundary tie count #{c < v} and #{c <= v}
__global__ void tau_tie_setup_kernel(TauArgs a) {
  if (threadIdx.x != 0) return;
  TauState &s = *a.st;
  for (int i = 0; i < a.n_q; ++i) {
    s.lo[i] = s.job[2 * i].prefix;
    s.hi[i] = s.job[2 * i + 1].prefix;
    s.mode[i] = (s.job[2 * i].active && s.lo[i] == s.hi[i]) ? 1 : 0;
    s.job[2 * i].active = 0;
    s.job[2 * i + 1].active = 0;
  }
}

__global__ __launch_bounds__(256) void tau_tie_count_kernel(TauArgs a) {
  __shared__ uint32_t v[kTauMaxQ];
  __shared__ int tie[kTauMaxQ];
  if (threadIdx.x < kTauMaxQ) {
    const bool on = threadIdx.x < a.n_q && a.st->mode[threadIdx.x] == 1;
    tie[threadIdx.x] = on ? 1 : 0;
    v[threadIdx.x] = on ? a.st->lo[threadIdx.x] : 0u;
  }
  __syncthreads();
  unsigned long long bl[kTauMaxQ], ab[kTauMaxQ];
#pragma unroll
  for (int i = 0; i < kTauMaxQ; ++i) bl[i] = ab[i] = 0ull;
  for (long long r = blockIdx.x * 256ll + threadIdx.x; r < a.n_rows; r += 256ll * gridDim.x) {
    float c[kMaxK];
    load_row(a, r, c);
    const unsigned cand = row_candidates(c, a.k, a.m_min);
#pragma unroll
    for (int i = 1; i < kMaxK; ++i) {
      if (!((cand >> i) & 1u)) continue;
      const uint32_t key = key_of(c[i]);
#pragma unroll
      for (int q = 0; q < kTauMaxQ; ++q) {
        bl[q] += (tie[q] && key < v[q]) ? 1ull : 0ull;
        ab[q] += (tie[q] && key <= v[q]) ? 1ull : 0ull;
      }
    }
  }
#pragma unroll
  for (int q = 0; q < kTauMaxQ; ++q) {
    const unsigned long long sb = block_sum(bl[q]);
    const unsigned long long sa = block_sum(ab[q]);
    if (threadIdx.x == 0 && tie[q]) {
      if (sb) atomicAdd(&a.st->below[q], sb);
      if (sa) atomicAdd(&a.st->above[q], sa);
    }
  }
}

// choose the side of a tied boundary; the midpoint side needs the next larger score
__global__ void tau_tie_choose_kernel(TauArgs a) {
  if (threadIdx.x != 0) return;
  TauState &s = *a.st;
  for (int i = 0; i < a.n_q; ++i) {
    if (s.mode[i] != 1) continue;
    const long long m = s.m_q[i];
    const long long below = static_cast<long long>(s.below[i]), above = static_cast<long long>(s.above[i]);
    const long long db = below > m ? below - m : m - below;
    const long long da = above > m ? above - m : m - above;
    if (db <= da) continue;                                   // tau = v
    if (above == static_cast<long long>(s.n_cand)) {
      s.mode[i] = 3;                                          // every candidate skipped
    } else {
      s.mode[i] = 2;
      s.job[2 * i] = Job{static_cast<unsigned long long>(above), 0u, 1};
    }
  }
}

__global__ void tau_finalize_kernel(TauArgs a) {
  if (threadIdx.x != 0) return;
  TauState &s = *a.st;
  const long long nc = static_cast<long long>(s.n_cand);
  for (int i = 0; i < a.n_q; ++i) {
    const long long m = s.m_q[i];
    float t;
    if (m == 0) {
      t = 0.f;
    } else if (m == nc) {
      t = INFINITY;
    } else if (s.mode[i] == 0) {
      t = static_cast<float>(0.5 * (static_cast<double>(value_of(s.lo[i])) + static_cast<double>(value_of(s.hi[i]))));
    } else if (s.mode[i] == 1) {
      t = value_of(s.lo[i]);
    } else if (s.mode[i] == 2) {
      t = static_cast<float>(0.5 * (static_cast<double>(value_of(s.lo[i])) +
                                    static_cast<double>(value_of(s.job[2 * i].prefix))));
    } else {
      t = INFINITY;
    }
    a.tau[i] = t;
    if (a.m_q_out) a.m_q_out[i] = m;
  }
  if (a.n_cand_out) a.n_cand_out[0] = nc;
}

void radix_select(const TauArgs &a, unsigned grid, hipStream_t stream) {
  for (int pass = 0; pass < 4; ++pass) {
    tau_hist_kernel<<<grid, 256, 0, stream>>>(a, pass);
    tau_pick_kernel<<<kJobs, kBins, 0, stream>>>(a, pass);
  }
}

}  // namespace

size_t tau_workspace_bytes() {
  return ((sizeof(TauState) + 255) / 256) * 256 + static_cast<size_t>(kJobs) * kBins * sizeof(unsigned long long);
}

hipError_t launch_tau_map(const float *scores, long long n_rows, int k, int m_min, const double *q, int n_q,
                          float *tau, long long *m_q_out, long long *n_cand_out, void *workspace,
                          hipStream_t stream) {
  TauArgs a{};
  a.scores = scores;
  a.n_rows = n_rows;
  a.k = k;
  a.m_min = m_min;
  a.n_q = n_q;
  for (int i = 0; i < kTauMaxQ; ++i) a.q[i] = i < n_q ? q[i] : 0.0;
  char *ws = static_cast<char *>(workspace);
  a.st = reinterpret_cast<TauState *>(ws);
  a.hist = reinterpret_cast<unsigned long long *>(ws + ((sizeof(TauState) + 255) / 256) * 256);
  a.tau = tau;
  a.m_q_out = m_q_out;
  a.n_cand_out = n_cand_out;
  long long blocks = (n_rows + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  const unsigned grid = static_cast<unsigned>(blocks);
  tau_init_kernel<<<1, 256, 0, stream>>>(a);
  tau_count_kernel<<<grid, 256, 0, stream>>>(a);
  tau_setup_kernel<<<1, 64, 0, stream>>>(a);
  radix_select(a, grid, stream);
  tau_tie_setup_kernel<<<1, 64, 0, stream>>>(a);
  tau_tie_count_kernel<<<grid, 256, 0, stream>>>(a);
  tau_tie_choose_kernel<<<1, 64, 0, stream>>>(a);
  radix_select(a, grid, stream);
  tau_finalize_kernel<<<1, 64, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace ace
