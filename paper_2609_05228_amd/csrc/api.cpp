// C ABI of the ACE MoE layer: host-side validation, workspace layout and the
// launch sequence of one layer forward (Alg. 1's online loop for one layer):
//   route (RMSNorm, router, top-k, Alg. 4 skip mask, per-chunk expert counts)
//   -> plan (expert scan, then prefix sum, permutation and M tiles)
//   -> grouped gate/up + SwiGLU -> grouped down
//   -> [shared expert: dense gate/up -> dense down] -> gate-weighted combine.
// Everything is enqueued on the caller's stream; nothing is allocated (the
// no-allocation variant runs in a static per-device scratch array instead of a
// caller workspace).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>
#include <vector>

#include "../../include/ace.h"
#include "ace_internal.h"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

constexpr int kSkinnyMaxT = 64;      // batches up to this many tokens take the small-batch GEMMs
constexpr long kSkinnyWaves = 4096;  // K-split until about this many waves stream weights

// K splits for the small-batch GEMMs: double while the work items stay under
// kSkinnyWaves and each split keeps a whole number of >= 2 64-wide K steps
int pick_splits(long items, int K) {
  int s = 1;
  while (s < 8 && items * s * 2 <= kSkinnyWaves && (K / (2 * s)) % 64 == 0 && K / (2 * s) >= 128 &&
         K % (2 * s) == 0)
    s *= 2;
  return s;
}

struct Layout {
  size_t xn, zpart, sspart, local_rank, chunk_count, chunk_base, slot_row, gates, counts, offsets, perm;
  size_t tile_e, tile_r0, tile_rows, tile_ord, n_tiles, H, Y, Hs, Ys, part_g, part_u, part_y, total;
  int G, max_groups, dense_groups;
  bool skinny;          // small-batch path (bf16, T <= kSkinnyMaxT)
  int splits_gu, splits_dn;
  int ksplit, zstride;  // router K slices (0: fused) and partial-logit row stride
};

Layout layout_for(const ace_moe_desc &d) {
  Layout L{};
  const size_t T = static_cast<size_t>(d.T), dd = static_cast<size_t>(d.d);
  const size_t N = static_cast<size_t>(d.N), k = static_cast<size_t>(d.k), m = static_cast<size_t>(d.m);
  const size_t esz = (d.dtype == ACE_BF16) ? 2 : 4;
  const size_t slots = T * k;
  L.G = static_cast<int>((T + ace::kRouteTokens - 1) / ace::kRouteTokens);
  // router: small batches spread W_r over (chunk, K slice) workgroups
  L.ksplit = 0;
  if (L.G <= ace::kRouteMaxSplitChunks) {
    const int nb = d.d / 32;
    L.ksplit = 1;
    while (L.ksplit < ace::kRouteMaxSlices && nb % (2 * L.ksplit) == 0 && L.G * L.ksplit < 128) L.ksplit *= 2;
  }
  L.zstride = 16 * ace::route_expert_tiles(d.N);
  L.skinny = d.dtype == ACE_BF16 && d.T <= kSkinnyMaxT;
  L.splits_gu = L.splits_dn = 1;
  if (L.skinny) {
    const long tiles = static_cast<long>(slots < N ? slots : N);
    L.splits_gu = pick_splits(tiles * (d.m / 16), d.d);
    L.splits_dn = pick_splits(tiles * (d.d / 32), d.m);
  }
  L.max_groups = static_cast<int>((slots + ace::kTileM - 1) / ace::kTileM + (slots < N ? slots : N));
  L.dense_groups = static_cast<int>((T + ace::kTileM - 1) / ace::kTileM);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.xn = take(T * dd * esz);
  L.zpart = take(static_cast<size_t>(L.ksplit) * T * L.zstride * 4);
  L.sspart = take(static_cast<size_t>(L.ksplit) * T * 4);
  L.local_rank = take(slots);
  L.chunk_count = take(static_cast<size_t>(L.G) * N);
  L.chunk_base = take(static_cast<size_t>(L.G) * N * 4);
  L.slot_row = take(slots * 4);
  L.gates = take(slots * 4);
  L.counts = take(N * 4);
  L.offsets = take((N + 1) * 4);
  L.perm = take(slots * 4);
  L.tile_e = take(static_cast<size_t>(L.max_groups) * 4);
  L.tile_r0 = take(static_cast<size_t>(L.max_groups) * 4);
  L.tile_rows = take(static_cast<size_t>(L.max_groups) * 4);
  L.tile_ord = take(static_cast<size_t>(L.max_groups) * 4);
  L.n_tiles = take(4);
  L.H = take(slots * m * esz);
  L.Y = take(slots * dd * esz);
  if (d.n_shared > 0) {
    L.Hs = take(T * static_cast<size_t>(d.m_shared) * esz);
    L.Ys = take(T * dd * esz);
  }
  if (L.splits_gu > 1) {
    L.part_g = take(static_cast<size_t>(L.splits_gu) * slots * m * 4);
    L.part_u = take(static_cast<size_t>(L.splits_gu) * slots * m * 4);
  }
  if (L.splits_dn > 1) L.part_y = take(static_cast<size_t>(L.splits_dn) * slots * dd * 4);
  L.total = off;
  return L;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

ace_status validate(const ace_moe_desc *d, const void *x, const ace_moe_weights *w,
                    const ace_moe_outputs *o) {
  if (!d || !w || !o) return ACE_ERR_INVALID_ARG;
  if (d->T < 0 || d->d <= 0 || d->N <= 0 || d->k <= 0 || d->m <= 0) return ACE_ERR_INVALID_ARG;
  if (d->k > d->N || d->m_min < 1 || d->m_min > d->k) return ACE_ERR_INVALID_ARG;
  if (d->dtype != ACE_F32 && d->dtype != ACE_BF16) return ACE_ERR_INVALID_ARG;
  if (d->n_shared < 0 || d->n_shared > 1) return ACE_ERR_INVALID_ARG;
  if (d->n_shared == 1 && d->m_shared <= 0) return ACE_ERR_INVALID_ARG;
  if (std::isnan(d->tau) || !std::isfinite(d->eps) || d->eps < 0.f || !std::isfinite(d->rms_eps) ||
      d->rms_eps < 0.f)
    return ACE_ERR_INVALID_ARG;
  if (d->flags & ~static_cast<uint32_t>(ACE_SKIP_DISABLE | ACE_WRITE_SCORES | ACE_FUSION_MASK))
    return ACE_ERR_INVALID_ARG;
  if (((d->flags & ACE_FUSION_MASK) >> ACE_FUSION_SHIFT) > ACE_FUSION_SCORE) return ACE_ERR_INVALID_ARG;
  if (d->N > ace::kMaxN || d->k > ace::kMaxK || d->d % 128 != 0 || d->m % 64 != 0 || d->d > 16384)
    return ACE_ERR_UNSUPPORTED;
  if (d->n_shared == 1 && d->m_shared % 64 != 0) return ACE_ERR_UNSUPPORTED;
  if (static_cast<int64_t>(d->T) * d->k >= (int64_t{1} << 31)) return ACE_ERR_UNSUPPORTED;
  if (d->T == 0) return ACE_OK;
  const void *req[] = {x, w->gamma, w->w_router, w->w_gate, w->w_up, w->w_down, w->a_gsp, w->a_rcr,
                       o->y, o->topk_idx, o->keep};
  for (const void *p : req)
    if (!p || !aligned16(p)) return ACE_ERR_INVALID_ARG;
  if (d->n_shared == 1) {
    const void *sreq[] = {w->ws_gate, w->ws_up, w->ws_down};
    for (const void *p : sreq)
      if (!p || !aligned16(p)) return ACE_ERR_INVALID_ARG;
  }
  const void *opt[] = {w->b_router, o->gates, o->scores, o->expert_counts, o->expert_offsets, o->perm};
  for (const void *p : opt)
    if (p && !aligned16(p)) return ACE_ERR_INVALID_ARG;
  if ((d->flags & ACE_WRITE_SCORES) && !o->scores) return ACE_ERR_INVALID_ARG;
  return ACE_OK;
}

// ---------------------------------------------------------------- stage timing
// Measurement hook only: while a profile is open, every forward records
// ACE_PROFILE_STAGES + 1 events on its stream (before the first stage and after
// each stage), one set per call, up to the capacity given at begin.
struct Profile {
  std::mutex mu;
  bool on = false;
  bool span = false;  // record only the first and the last event of each call
  int cap = 0;
  int used = 0;
  std::vector<hipEvent_t> ev;  // cap x (stages + 1)
  std::vector<uint8_t> rec;    // cap x (stages + 1): event recorded (a stage that launches nothing records none)
};
Profile g_prof;
constexpr int kStages = ACE_PROFILE_STAGES;

// events of the next call, or null when no profile is open (or it is full)
struct ProfSlot {
  hipEvent_t *ev = nullptr;
  uint8_t *rec = nullptr;
  bool span = false;
};
ProfSlot profile_slot() {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || g_prof.used >= g_prof.cap) return {};
  const size_t o = static_cast<size_t>(g_prof.used++) * (kStages + 1);
  std::fill(g_prof.rec.begin() + o, g_prof.rec.begin() + o + kStages + 1, uint8_t{0});
  return {&g_prof.ev[o], &g_prof.rec[o], g_prof.span};
}

// event i after stage i-1; `launched` = false for a stage that enqueued nothing, whose
// time then counts as zero (each record costs the stream a few microseconds)
void mark(const ProfSlot &slot, int i, hipStream_t s, bool launched = true) {
  if (slot.ev && ((launched && !slot.span) || i == 0 || i == kStages)) {
    (void)hipEventRecord(slot.ev[i], s);
    slot.rec[i] = 1;
  }
}

// ---------------------------------------------------------------- static scratch
// Workspace of ace_moe_forward_noalloc: one array per GPU, part of this library's
// code object (each GPU holds its own copy from the first use until the process
// ends).  In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device with hipGetSymbolAddress and only
// that address is ever handed to kernels.
static __device__ __align__(256) uint8_t scratch[ACE_NOALLOC_SCRATCH_BYTES];

struct ScratchTable {
  std::mutex mu;
  std::vector<void *> ptr;  // device id -> address of that device's scratch (null: not yet looked up)
};
ScratchTable g_scratch;

// address of the current device's scratch, looked up (with that device current) on
// the first call on the device
hipError_t scratch_on_current_device(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch.mu);
  if (static_cast<size_t>(dev) >= g_scratch.ptr.size()) g_scratch.ptr.resize(static_cast<size_t>(dev) + 1, nullptr);
  if (!g_scratch.ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (reinterpret_cast<uintptr_t>(p) & (kAlign - 1))) return hipErrorInvalidSymbol;
    g_scratch.ptr[dev] = p;
  }
  *out = g_scratch.ptr[dev];
  return hipSuccess;
}

ace_status profile_open(int max_calls, bool span) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (g_prof.on || max_calls <= 0 || max_calls > 100000) return ACE_ERR_INVALID_ARG;
  g_prof.ev.assign(static_cast<size_t>(max_calls) * (kStages + 1), nullptr);
  // timing-only events: no system-scope fence when recorded, so recording one does not
  // write back and invalidate the caches between the stages it separates (a fenced
  // record costs the stream several microseconds)
  for (auto &e : g_prof.ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) {
      for (auto &x : g_prof.ev)
        if (x) (void)hipEventDestroy(x);
      g_prof.ev.clear();
      return ACE_ERR_HIP;
    }
  g_prof.rec.assign(g_prof.ev.size(), uint8_t{0});
  g_prof.cap = max_calls;
  g_prof.used = 0;
  g_prof.span = span;
  g_prof.on = true;
  return ACE_OK;
}

ace_status forward_impl(const ace_moe_desc *desc, const void *x, const ace_moe_weights *w,
                        const ace_moe_outputs *out, void *workspace, size_t workspace_bytes,
                        void *stream_ptr);

}  // namespace

extern "C" {

ace_status ace_profile_begin(int max_calls) { return profile_open(max_calls, false); }

ace_status ace_profile_begin_span(int max_calls) { return profile_open(max_calls, true); }

ace_status ace_profile_end(double *stage_ms, int n_stages, int *n_calls, double *call_stage_ms, int max_calls) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on) return ACE_ERR_INVALID_ARG;
  ace_status st = ACE_OK;
  for (int j = 0; j < n_stages && stage_ms; ++j) stage_ms[j] = 0.0;
  for (int c = 0; c < g_prof.used && st == ACE_OK; ++c) {
    hipEvent_t *e = &g_prof.ev[static_cast<size_t>(c) * (kStages + 1)];
    const uint8_t *rec = &g_prof.rec[static_cast<size_t>(c) * (kStages + 1)];
    if (hipEventSynchronize(e[kStages]) != hipSuccess) {
      st = ACE_ERR_HIP;
      break;
    }
    // stage j spans the last recorded event at or before j to event j+1; a stage whose
    // end event was not recorded enqueued nothing and counts zero
    int last = 0;
    for (int j = 0; j < kStages; ++j) {
      float ms = 0.f;
      if (rec[j + 1]) {
        if (hipEventElapsedTime(&ms, e[last], e[j + 1]) != hipSuccess) {
          st = ACE_ERR_HIP;
          break;
        }
        last = j + 1;
      }
      if (j < n_stages) {
        if (stage_ms) stage_ms[j] += ms;
        if (call_stage_ms && c < max_calls) call_stage_ms[static_cast<size_t>(c) * n_stages + j] = ms;
      }
    }
  }
  if (n_calls) *n_calls = g_prof.used;
  for (auto &x : g_prof.ev) (void)hipEventDestroy(x);
  g_prof.ev.clear();
  g_prof.rec.clear();
  g_prof.on = false;
  g_prof.span = false;
  g_prof.cap = g_prof.used = 0;
  return st;
}


size_t ace_moe_workspace_size(const ace_moe_desc *desc) {
  if (!desc || desc->T <= 0 || desc->d <= 0 || desc->N <= 0 || desc->k <= 0 || desc->m <= 0) return 0;
  return layout_for(*desc).total;
}

int ace_abi_version(void) { return ACE_ABI_VERSION; }

size_t ace_tables_workspace_size(const ace_moe_desc *desc) {
  if (!desc || desc->N <= 0 || desc->d <= 0 || desc->m <= 0) return 0;
  return ace::tables_workspace_bytes(desc->N, desc->d, desc->m);
}

ace_status ace_build_tables(const ace_moe_desc *desc, const ace_moe_weights *w, float *a_gsp, float *a_rcr,
                            double *a_gsp64, double *a_rcr64, void *workspace, size_t workspace_bytes,
                            void *stream) {
  if (!desc || !w || !a_gsp || !a_rcr) return ACE_ERR_INVALID_ARG;
  const ace_moe_desc &d = *desc;
  if (d.N <= 0 || d.d <= 0 || d.m <= 0 || (d.dtype != ACE_F32 && d.dtype != ACE_BF16) || !(d.eps >= 0.f))
    return ACE_ERR_INVALID_ARG;
  if (d.m % 64 != 0 || d.d % 32 != 0) return ACE_ERR_UNSUPPORTED;
  const size_t align = 16;  // 16-byte operand loads
  const void *need[] = {w->gamma, w->w_router, w->w_gate, w->w_up, w->w_down};
  for (const void *p : need)
    if (!p || (reinterpret_cast<uintptr_t>(p) & (align - 1))) return ACE_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(a_gsp) & 3) || (reinterpret_cast<uintptr_t>(a_rcr) & 3) ||
      (reinterpret_cast<uintptr_t>(a_gsp64) & 7) || (reinterpret_cast<uintptr_t>(a_rcr64) & 7))
    return ACE_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < ace::tables_workspace_bytes(d.N, d.d, d.m) ||
      (reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)))
    return ACE_ERR_WORKSPACE;
  ace::TablesCall c{};
  c.gamma = w->gamma;
  c.w_router = w->w_router;
  c.w_gate = w->w_gate;
  c.w_up = w->w_up;
  c.w_down = w->w_down;
  c.N = d.N;
  c.d = d.d;
  c.m = d.m;
  c.eps = d.eps;
  c.bf16 = d.dtype == ACE_BF16;
  c.workspace = workspace;
  c.a_gsp = a_gsp;
  c.a_rcr = a_rcr;
  c.a_gsp64 = a_gsp64;
  c.a_rcr64 = a_rcr64;
  return ace::launch_tables(c, static_cast<hipStream_t>(stream)) == hipSuccess ? ACE_OK : ACE_ERR_HIP;
}

size_t ace_tau_workspace_size(void) { return ace::tau_workspace_bytes(); }

ace_status ace_tau_map(const float *scores, int64_t n_rows, int32_t k, int32_t m_min, const double *q,
                       int32_t n_q, float *tau, int64_t *m_q, int64_t *n_cand, void *workspace,
                       size_t workspace_bytes, void *stream) {
  static_assert(ACE_TAU_MAX_Q == ace::kTauMaxQ, "tau budget count");
  if (k < 1 || k > ace::kMaxK || m_min < 1 || m_min > k || n_rows < 0 || n_q < 1 || n_q > ACE_TAU_MAX_Q)
    return ACE_ERR_INVALID_ARG;
  if (!q || !tau || (n_rows > 0 && !scores)) return ACE_ERR_INVALID_ARG;
  if (n_rows > (static_cast<int64_t>(1) << 40)) return ACE_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(scores) & 3) || (reinterpret_cast<uintptr_t>(tau) & 3) ||
      (reinterpret_cast<uintptr_t>(m_q) & 7) || (reinterpret_cast<uintptr_t>(n_cand) & 7))
    return ACE_ERR_INVALID_ARG;
  for (int i = 0; i < n_q; ++i)
    if (!(q[i] >= 0.0 && q[i] <= 1.0)) return ACE_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < ace::tau_workspace_bytes() ||
      (reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)))
    return ACE_ERR_WORKSPACE;
  const hipError_t e = ace::launch_tau_map(scores, n_rows, k, m_min, q, n_q, tau, reinterpret_cast<long long *>(m_q),
                                           reinterpret_cast<long long *>(n_cand), workspace,
                                           static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACE_OK : ACE_ERR_HIP;
}

const char *ace_status_string(int s) {
  switch (s) {
    case ACE_OK: return "ACE_OK: success";
    case ACE_ERR_INVALID_ARG: return "ACE_ERR_INVALID_ARG: invalid argument (NULL, shape, alignment or scalar)";
    case ACE_ERR_UNSUPPORTED: return "ACE_ERR_UNSUPPORTED: shape or dtype outside the compiled set";
    case ACE_ERR_WORKSPACE: return "ACE_ERR_WORKSPACE: workspace missing or too small";
    case ACE_ERR_HIP: return "ACE_ERR_HIP: a HIP launch failed";
    case ACE_ERR_SCRATCH_LIMIT:
      return "ACE_ERR_SCRATCH_LIMIT: the layer needs more than the ACE_NOALLOC_SCRATCH_BYTES of static scratch "
             "(use ace_moe_forward with a workspace)";
    default: return "unknown ace_status";
  }
}

ace_status ace_moe_forward(const ace_moe_desc *desc, const void *x, const ace_moe_weights *w,
                           const ace_moe_outputs *out, void *workspace, size_t workspace_bytes,
                           void *stream_ptr) {
  return forward_impl(desc, x, w, out, workspace, workspace_bytes, stream_ptr);
}

ace_status ace_moe_forward_noalloc(const ace_moe_desc *desc, const void *x, const ace_moe_weights *w,
                                   const ace_moe_outputs *out, void *stream_ptr) {
  const ace_status v = validate(desc, x, w, out);
  if (v != ACE_OK) return v;
  if (desc->T == 0) return ACE_OK;
  const size_t need = layout_for(*desc).total;
  if (need > ACE_NOALLOC_SCRATCH_BYTES) return ACE_ERR_SCRATCH_LIMIT;
  void *ws = nullptr;
  if (scratch_on_current_device(&ws) != hipSuccess) return ACE_ERR_HIP;
  return forward_impl(desc, x, w, out, ws, ACE_NOALLOC_SCRATCH_BYTES, stream_ptr);
}

}  // extern "C"

namespace {

ace_status forward_impl(const ace_moe_desc *desc, const void *x, const ace_moe_weights *w,
                        const ace_moe_outputs *out, void *workspace, size_t workspace_bytes,
                        void *stream_ptr) {
  const ace_status v = validate(desc, x, w, out);
  if (v != ACE_OK) return v;
  const ace_moe_desc &d = *desc;
  if (d.T == 0) return ACE_OK;
  const Layout L = layout_for(d);
  if (!workspace || workspace_bytes < L.total || (reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)))
    return ACE_ERR_WORKSPACE;

  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  char *ws = static_cast<char *>(workspace);
  const bool bf16 = d.dtype == ACE_BF16;
  auto at = [&](size_t off) { return static_cast<void *>(ws + off); };

  auto *local_rank = static_cast<uint8_t *>(at(L.local_rank));
  auto *chunk_count = static_cast<uint8_t *>(at(L.chunk_count));
  auto *chunk_base = static_cast<int32_t *>(at(L.chunk_base));
  auto *slot_row = static_cast<int32_t *>(at(L.slot_row));
  float *gates = out->gates ? out->gates : static_cast<float *>(at(L.gates));
  int32_t *counts = out->expert_counts ? out->expert_counts : static_cast<int32_t *>(at(L.counts));
  int32_t *offsets = out->expert_offsets ? out->expert_offsets : static_cast<int32_t *>(at(L.offsets));
  int32_t *perm = out->perm ? out->perm : static_cast<int32_t *>(at(L.perm));
  auto *tile_e = static_cast<int32_t *>(at(L.tile_e));
  auto *tile_r0 = static_cast<int32_t *>(at(L.tile_r0));
  auto *tile_rows = static_cast<int32_t *>(at(L.tile_rows));
  auto *tile_ord = static_cast<int32_t *>(at(L.tile_ord));
  auto *n_tiles = static_cast<int32_t *>(at(L.n_tiles));

  const ProfSlot prof = profile_slot();
  mark(prof, 0, stream);

  ace::RouteArgs ra{};
  ra.x = x;
  ra.gamma = w->gamma;
  ra.w_router = w->w_router;
  ra.b_router = w->b_router;
  ra.a_gsp = w->a_gsp;
  ra.a_rcr = w->a_rcr;
  ra.xn = at(L.xn);
  ra.topk_idx = out->topk_idx;
  ra.keep = out->keep;
  ra.gates = gates;
  ra.scores = (d.flags & ACE_WRITE_SCORES) ? out->scores : nullptr;
  ra.slot_row = slot_row;
  ra.local_rank = local_rank;
  ra.chunk_count = chunk_count;
  ra.zpart = static_cast<float *>(at(L.zpart));
  ra.sspart = static_cast<float *>(at(L.sspart));
  ra.ksplit = L.ksplit;
  ra.counts = counts;
  ra.offsets = offsets;
  ra.perm = perm;
  ra.tile_expert = tile_e;
  ra.tile_row0 = tile_r0;
  ra.tile_rows = tile_rows;
  ra.n_tiles = n_tiles;
  ra.zstride = L.zstride;
  ra.T = d.T;
  ra.d = d.d;
  ra.N = d.N;
  ra.k = d.k;
  ra.m_min = d.m_min;
  ra.tau = d.tau;
  ra.eps = d.eps;
  ra.rms_eps = d.rms_eps;
  ra.skip_disable = (d.flags & ACE_SKIP_DISABLE) ? 1 : 0;
  ra.fusion = static_cast<int>((d.flags & ACE_FUSION_MASK) >> ACE_FUSION_SHIFT);
  if (ace::launch_route(ra, bf16, stream) != hipSuccess) return ACE_ERR_HIP;
  mark(prof, 1, stream);

  ace::PlanArgs pa{};
  pa.chunk_count = chunk_count;
  pa.local_rank = local_rank;
  pa.topk_idx = out->topk_idx;
  pa.keep = out->keep;
  pa.chunk_base = chunk_base;
  pa.counts = counts;
  pa.offsets = offsets;
  pa.perm = perm;
  pa.slot_row = slot_row;
  pa.tile_expert = tile_e;
  pa.tile_row0 = tile_r0;
  pa.tile_rows = tile_rows;
  pa.tile_order = tile_ord;
  pa.n_tiles = n_tiles;
  pa.T = d.T;
  pa.k = d.k;
  pa.N = d.N;
  pa.G = L.G;
  // one chunk: the router's select workgroup already wrote the plan; several chunks of a
  // small bf16 batch: the skinny gate/up kernel derives it (SkinnyArgs::self_plan)
  const bool self_plan = L.skinny && L.G > 1;
  const bool planned = (L.ksplit > 0 && L.G == 1) || self_plan;
  if (!planned && ace::launch_plan(pa, stream) != hipSuccess) return ACE_ERR_HIP;
  mark(prof, 2, stream, !planned);

  ace::GemmArgs g{};
  g.act = at(L.xn);
  g.perm = perm;
  g.w0 = w->w_gate;
  g.w1 = w->w_up;
  g.out = at(L.H);
  g.tile_expert = tile_e;
  g.tile_row0 = tile_r0;
  g.tile_rows = tile_rows;
  g.n_tiles = n_tiles;
  // the gate/up launch takes the plan kernel's tile order when it wrote one
  g.tile_order = (!planned && ace::plan_writes_order(pa)) ? tile_ord : nullptr;
  g.dense_rows = 0;
  g.max_groups = L.max_groups;
  g.d = d.d;
  g.m = d.m;
  ace::GemmArgs gd = g;
  gd.tile_order = nullptr;  // the down launch keeps list order
  gd.act = at(L.H);
  gd.perm = nullptr;
  gd.w0 = w->w_down;
  gd.w1 = nullptr;
  gd.out = at(L.Y);
  // a shared expert with the routed experts' intermediate size runs as extra M tiles
  // of the routed grouped GEMMs (one launch each instead of two half-filled ones)
  const bool shared_in_routed = d.n_shared == 1 && bf16 && !L.skinny && d.m_shared == d.m;
  if (shared_in_routed) {
    const int st = L.dense_groups;
    g.sh_tiles = gd.sh_tiles = st;
    g.sh_rows = gd.sh_rows = d.T;
    g.max_groups += st;
    gd.max_groups += st;
    g.sh_act = at(L.xn);
    g.sh_w0 = w->ws_gate;
    g.sh_w1 = w->ws_up;
    g.sh_out = at(L.Hs);
    gd.sh_act = at(L.Hs);
    gd.sh_w0 = w->ws_down;
    gd.sh_w1 = nullptr;
    gd.sh_out = at(L.Ys);
  }
  if (L.skinny) {
    const int slots = d.T * d.k;
    ace::SkinnyArgs su{g, L.splits_gu, slots, static_cast<float *>(at(L.part_g)), static_cast<float *>(at(L.part_u))};
    if (self_plan) {
      su.self_plan = true;
      su.topk_idx = out->topk_idx;
      su.keep = out->keep;
      su.chunk_count = chunk_count;
      su.counts = counts;
      su.offsets = offsets;
      su.perm = perm;
      su.slot_row = slot_row;
      su.tile_expert = tile_e;
      su.tile_row0 = tile_r0;
      su.tile_rows = tile_rows;
      su.n_tiles = n_tiles;
      su.T = d.T;
      su.k = d.k;
      su.N = d.N;
      su.G = L.G;
    }
    if (ace::launch_skinny(su, true, offsets + d.N, stream) != hipSuccess) return ACE_ERR_HIP;
    mark(prof, 3, stream);
    ace::SkinnyArgs sd{gd, L.splits_dn, slots, static_cast<float *>(at(L.part_y)), nullptr};
    if (ace::launch_skinny(sd, false, offsets + d.N, stream) != hipSuccess) return ACE_ERR_HIP;
  } else {
    if (ace::launch_gateup(g, bf16, stream) != hipSuccess) return ACE_ERR_HIP;
    mark(prof, 3, stream);
    if (ace::launch_down(gd, bf16, stream) != hipSuccess) return ACE_ERR_HIP;
  }
  mark(prof, 4, stream);

  const void *Ys = shared_in_routed ? at(L.Ys) : nullptr;
  if (d.n_shared == 1 && !shared_in_routed) {
    ace::GemmArgs s{};
    s.act = at(L.xn);
    s.perm = nullptr;
    s.w0 = w->ws_gate;
    s.w1 = w->ws_up;
    s.out = at(L.Hs);
    s.dense_rows = d.T;
    s.max_groups = L.dense_groups;
    s.d = d.d;
    s.m = d.m_shared;
    ace::GemmArgs sd = s;
    sd.act = at(L.Hs);
    sd.w0 = w->ws_down;
    sd.w1 = nullptr;
    sd.out = at(L.Ys);
    if (L.skinny) {
      ace::SkinnyArgs su{s, 1, d.T, nullptr, nullptr};
      ace::SkinnyArgs sdn{sd, 1, d.T, nullptr, nullptr};
      if (ace::launch_skinny(su, true, nullptr, stream) != hipSuccess) return ACE_ERR_HIP;
      if (ace::launch_skinny(sdn, false, nullptr, stream) != hipSuccess) return ACE_ERR_HIP;
    } else {
      if (ace::launch_gateup(s, bf16, stream) != hipSuccess) return ACE_ERR_HIP;
      if (ace::launch_down(sd, bf16, stream) != hipSuccess) return ACE_ERR_HIP;
    }
    Ys = at(L.Ys);
  }
  mark(prof, 5, stream, d.n_shared == 1 && !shared_in_routed);

  ace::CombineArgs c{};
  c.Y = at(L.Y);
  c.Ypart = L.splits_dn > 1 ? static_cast<const float *>(at(L.part_y)) : nullptr;
  c.ysplits = L.splits_dn;
  c.rows_cap = d.T * d.k;
  c.Ys = Ys;
  c.slot_row = slot_row;
  c.gates = gates;
  c.y = out->y;
  c.T = d.T;
  c.d = d.d;
  c.k = d.k;
  if (ace::launch_combine(c, bf16, stream) != hipSuccess) return ACE_ERR_HIP;
  mark(prof, 6, stream);
  return ACE_OK;
}

}  // namespace
