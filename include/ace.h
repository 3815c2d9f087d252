/*
 * ace.h — C ABI of the ACE token-adaptive MoE layer for AMD Instinct MI355X (gfx950).
 *
 * The library computes one MoE layer forward with ACE's calibration-free expert
 * skipping (arxiv 2609.05228): RMSNorm, router logits, softmax/top-k with gate
 * renormalisation, the ACE skip mask (Alg. 4, "ACE: Online Conservative Expert
 * Skipping"), and the sparsified output y_t = sum_{i in I_t} ghat_i f_{e_i}(x_t)
 * (Eq. ace_sparse_output), where f_e is the SwiGLU expert of Eq. swiglu_expert.
 * The per-expert GSP and RCR amplification tables (Alg. 2, Alg. 3) and the
 * threshold tau (App. C.1) are inputs: "per-expert statistics in, layer input and
 * weights in, output plus skip mask out".
 *
 * Conventions for every entry point
 *   - Pointers marked DEVICE are device (HBM) pointers; the caller owns every
 *     buffer.  The library allocates nothing and keeps no per-call state.
 *   - Descriptor, weight and output structs are HOST structs passed by pointer;
 *     they are read during the call only.
 *   - ace_moe_forward validates everything on the host before any launch; on an
 *     error nothing is enqueued and the returned status says why.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and the
 *     call returns without synchronising the host.
 *   - All arrays are dense row-major with the layouts stated below; every device
 *     pointer must be 16-byte aligned.
 */
#ifndef ACE_H
#define ACE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ACE_ABI_VERSION 5

typedef enum {
  ACE_OK = 0,
  ACE_ERR_INVALID_ARG = -1, /* NULL required pointer, bad shape, misaligned pointer, bad scalar */
  ACE_ERR_UNSUPPORTED = -2, /* valid but outside the compiled shape/dtype set (see ace_moe_forward) */
  ACE_ERR_WORKSPACE = -3,   /* workspace NULL or smaller than ace_moe_workspace_size() */
  ACE_ERR_HIP = -4,         /* a HIP launch reported an error */
  ACE_ERR_SCRATCH_LIMIT = -5 /* ace_moe_forward_noalloc: the layer needs more than its static scratch */
} ace_status;

typedef enum { ACE_F32 = 0, ACE_BF16 = 1 } ace_dtype;

enum {
  /* Plain top-k layer through the same kernels: every routed slot is kept and
     ghat = g exactly (no epsilon).  This is the unskipped baseline. */
  ACE_SKIP_DISABLE = 1u << 0,
  /* Fill outputs.scores with the contribution c of every routed slot (under the
     selected fusion rule; ACE: c = max(p_GSP, p_RCR), Eq. ace_contribution), as the
     App. C.1 score pass needs. */
  ACE_WRITE_SCORES = 1u << 1
};

/* Contribution rule, stored in flags bits 2-4 as (rule << ACE_FUSION_SHIFT).  A slot
   other than the top-1 is skippable iff c < tau; the m_min safeguard restores skipped
   slots by descending c.  ACE is the max rule (Alg. 4); the others are the variants
   the paper ablates (Tab. fusion_ablation, Tab. ablation) and its router-score
   baseline (Sec. 4.1).  p_GSP, p_RCR are Eqs. gsp_probability, rcr_probability. */
typedef enum {
  ACE_FUSION_MAX = 0,   /* c = max(p_GSP, p_RCR): skip only if both views are low      */
  ACE_FUSION_MIN = 1,   /* c = min(p_GSP, p_RCR): skip if either view is low (union)    */
  ACE_FUSION_MEAN = 2,  /* c = (p_GSP + p_RCR) / 2                                      */
  ACE_FUSION_GSP = 3,   /* c = p_GSP (single view)                                      */
  ACE_FUSION_RCR = 4,   /* c = p_RCR (single view)                                      */
  ACE_FUSION_SCORE = 5  /* c = g / (sum_j g_j + eps): router-score skipping, tables unused */
} ace_fusion;
#define ACE_FUSION_SHIFT 2
#define ACE_FUSION_MASK (7u << ACE_FUSION_SHIFT)

/* Layer shape and the scalars of Alg. 4. */
typedef struct {
  int32_t T;        /* tokens (0 = nothing to do) */
  int32_t d;        /* hidden size */
  int32_t N;        /* routed experts */
  int32_t k;        /* top-k */
  int32_t m;        /* expert intermediate size */
  int32_t n_shared; /* 0 or 1 ungated, always-active shared expert (not a routed slot) */
  int32_t m_shared; /* its intermediate size (ignored when n_shared = 0) */
  int32_t dtype;    /* ace_dtype of x, gamma, every weight matrix and y */
  int32_t m_min;    /* minimum active experts per token, 1..k (1 = top-1 safeguard only) */
  float tau;        /* threshold tau_q; a slot is skippable iff c < tau (strict) */
  float eps;        /* epsilon of Alg. 4 (both score normalisations and the gate renormalisation) */
  float rms_eps;    /* RMSNorm epsilon: x_in = x / sqrt(mean(x^2) + rms_eps) * gamma */
  uint32_t flags;   /* ACE_SKIP_DISABLE | ACE_WRITE_SCORES | (ace_fusion << ACE_FUSION_SHIFT) */
} ace_moe_desc;

/* Frozen layer parameters (DEVICE pointers, dtype = desc.dtype unless stated). */
typedef struct {
  const void *gamma;     /* [d]      RMSNorm scale (the diagonal of Gamma_l, Sec. 3.1)        */
  const void *w_router;  /* [N, d]   row e is the router vector w_e (Eq. app_router_logit)     */
  const float *b_router; /* [N] fp32 router bias b_e, or NULL for none                       */
  const void *w_gate;    /* [N, m, d] per-expert gate projection (nn.Linear out x in layout)  */
  const void *w_up;      /* [N, m, d] per-expert up projection                               */
  const void *w_down;    /* [N, d, m] per-expert down projection                             */
  const void *ws_gate;   /* [m_shared, d] shared-expert gate, or NULL when n_shared = 0       */
  const void *ws_up;     /* [m_shared, d]                                                    */
  const void *ws_down;   /* [d, m_shared]                                                    */
  const float *a_gsp;    /* [N] fp32 A^GSP(e), Alg. 2 output (Eq. gsp_layer_normalization)   */
  const float *a_rcr;    /* [N] fp32 A^RCR(e), Alg. 3 output (Eq. rcr_layer_normalization)   */
} ace_moe_weights;

/* Outputs (DEVICE pointers).  Required ones are fully overwritten; NULL optional
   ones are skipped. */
typedef struct {
  void *y;                 /* [T, d] dtype, required: the layer output (Eq. ace_sparse_output) */
  int32_t *topk_idx;       /* [T, k] required: routed experts in descending router probability;
                              equal logits go to the lower expert id; slot 0 is the top-1 expert */
  uint8_t *keep;           /* [T, k] required: 1 = slot in the active set I_t, 0 = skipped      */
  float *gates;            /* [T, k] optional: ghat (renormalised gate, 0 where skipped)        */
  float *scores;           /* [T, k] optional: c (written only with ACE_WRITE_SCORES)          */
  int32_t *expert_counts;  /* [N]    optional: kept slots per expert                          */
  int32_t *expert_offsets; /* [N+1]  optional: exclusive prefix sum of expert_counts          */
  int32_t *perm;           /* [T*k]  optional: token of each kept slot in (expert, token)
                              ascending order; entries past sum(expert_counts) are undefined */
} ace_moe_outputs;

/* Bytes of DEVICE scratch memory ace_moe_forward needs for `desc`
   (0 if desc is NULL or T <= 0).  Depends only on the shape fields and dtype. */
size_t ace_moe_workspace_size(const ace_moe_desc *desc);

/*
 * One ACE MoE layer forward (Alg. 1's online loop for one layer).
 *   x          DEVICE [T, d] layer input before RMSNorm, dtype = desc->dtype.
 *   workspace  DEVICE scratch of at least ace_moe_workspace_size(desc) bytes,
 *              256-byte aligned; its contents on entry do not matter.  Calls that
 *              share one workspace must be ordered on one stream.
 *   stream     hipStream_t to enqueue on (NULL = null stream).
 * Compiled shape set (else ACE_ERR_UNSUPPORTED): N <= 256, k <= 8, d % 128 == 0,
 * m % 64 == 0, m_shared % 64 == 0, d <= 16384, T * k < 2^31.
 * Semantics: tau <= 0 skips nothing (ghat = g / (1 + eps)); tau = +inf skips every
 * slot but the top-1 (and the m_min safeguard).  Skipped slots keep their topk_idx
 * entry and get keep = 0, ghat = 0.  Results are deterministic: two calls on the
 * same inputs give bit-identical outputs.
 */
ace_status ace_moe_forward(const ace_moe_desc *desc, const void *x, const ace_moe_weights *w,
                           const ace_moe_outputs *out, void *workspace, size_t workspace_bytes,
                           void *stream);

/*
 * ace_moe_forward without a workspace argument and without any allocation, for
 * callers that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Same arguments, semantics,
 * kernels and results as ace_moe_forward (bit-identical outputs), except that the
 * scratch memory is a static array of ACE_NOALLOC_SCRATCH_BYTES inside the
 * library's code object, one per GPU, which that GPU holds from the first call on
 * it until the process ends.  The call runs on the current device (the one
 * `stream` belongs to) and allocates nothing: no hipMalloc, no hipFree, no
 * allocating library routine.  The first call on a device looks up that device's
 * array address once (hipGetSymbolAddress; no allocation).
 *   Limit: layers whose ace_moe_workspace_size(desc) exceeds
 *   ACE_NOALLOC_SCRATCH_BYTES -> ACE_ERR_SCRATCH_LIMIT before any launch (for the
 *   d = 2048, N = 128, k = 8, m = 768 bf16 layer that is T above 1361 tokens;
 *   decode batches fit easily).
 *   Concurrency: every call on one GPU uses that GPU's one array, which keeps the
 *   last call's contents (no call depends on them).  Calls that can overlap on one
 *   GPU (different streams without ordering, or host threads racing on streams of
 *   the same device) race on the array and give wrong results; order them on one
 *   stream, or use ace_moe_forward with separate workspaces.
 * Errors: as ace_moe_forward, ACE_ERR_SCRATCH_LIMIT as above, ACE_ERR_HIP if the
 * device or its array cannot be found.
 */
#define ACE_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
ace_status ace_moe_forward_noalloc(const ace_moe_desc *desc, const void *x, const ace_moe_weights *w,
                                   const ace_moe_outputs *out, void *stream);

/*
 * Stage timing, for measurement only (computing the layer never needs it).
 * ace_profile_begin(max_calls) creates max_calls x (ACE_PROFILE_STAGES + 1) HIP
 * events on the current device; each following ace_moe_forward (up to max_calls)
 * records one set on its own stream: before the first stage and after each stage
 *   0 route  (RMSNorm, router, top-k, Alg. 4 skip mask, per-chunk expert counts)
 *   1 plan   (expert histogram and prefix sums, permutation, M tiles)
 *   2 gateup (grouped gate/up GEMM with the SwiGLU epilogue)
 *   3 down   (grouped down GEMM)
 *   4 shared (dense shared expert; empty when n_shared = 0)
 *   5 combine.
 * ace_profile_end waits for the recorded events, writes the per-stage elapsed
 * time summed over the recorded calls (ms) into stage_ms[0..n_stages-1] and the
 * number of recorded calls into *n_calls, optionally each call's stage times into
 * call_stage_ms[c * n_stages + j] for the first max_calls calls (NULL: not
 * written; the sum over j is that call's time from the start of its first stage
 * to the end of its last; a stage that enqueued nothing for the call, such as the
 * shared expert of a layer without one, records no event and counts zero), and
 * destroys the events.  The events are created
 * without a system-scope fence (timing only), so recording them does not flush
 * the caches between stages.  Only one profile may be open per process; begin
 * while open -> ACE_ERR_INVALID_ARG.
 * ace_profile_begin_span(max_calls) opens the same profile, but each call records
 * only its first and its last event: a call's time is the span of the whole layer
 * without the intermediate records (each one costs the stream about a
 * microsecond), and ace_profile_end reports all of it as the last stage's.
 */
#define ACE_PROFILE_STAGES 6
ace_status ace_profile_begin(int max_calls);
ace_status ace_profile_begin_span(int max_calls);
ace_status ace_profile_end(double *stage_ms, int n_stages, int *n_calls, double *call_stage_ms, int max_calls);

/*
 * Budget-to-threshold mapping (App. C.1) on the device.  From the contribution
 * scores of one unlabeled score pass (outputs.scores of ace_moe_forward with
 * ACE_WRITE_SCORES; any tau, the scores do not depend on it), computes for each
 * requested skip ratio q the threshold tau_q that realises it:
 *   N_all  = n_rows * k routed slots;
 *   N_cand = slots other than slot 0 (top-1) and, with m_min > 1, the m_min - 1
 *            highest-c other slots of each row (ties to the lower slot);
 *   m_q    = clip(round-half-even(q * N_all), 0, N_cand);
 *   tau_q  = midpoint of the m_q-th and (m_q+1)-th smallest candidate scores when
 *            they differ; on a tie at value v, v or the midpoint of v and the next
 *            larger score, whichever realises a count closer to m_q (the lower count
 *            on a draw); 0 when m_q = 0, +inf when m_q = N_cand.
 * A pass over several layers is one call over their scores stacked as rows (one
 * global tau per model).  With that tau, ace_moe_forward on the same inputs skips
 * exactly the candidates with c < tau_q.  Midpoints are formed in fp64 from the
 * fp32 scores and rounded once to fp32.
 *   scores     DEVICE [n_rows, k] fp32 (row r = one token of one layer, slot 0 = top-1);
 *              may be NULL when n_rows = 0.
 *   q          HOST [n_q] skip ratios in [0, 1]; 1 <= n_q <= ACE_TAU_MAX_Q.
 *   tau        DEVICE [n_q] fp32 out.
 *   m_q        DEVICE [n_q] int64 out, optional (NULL): the target skip counts.
 *   n_cand     DEVICE [1] int64 out, optional (NULL).
 *   workspace  DEVICE scratch of ace_tau_workspace_size() bytes, 256-byte aligned.
 * Enqueued on `stream` with no host synchronisation; deterministic.
 * Errors: k outside 1..8, m_min outside 1..k, n_rows < 0, n_q outside
 * 1..ACE_TAU_MAX_Q, q outside [0, 1] or NaN, NULL required pointers ->
 * ACE_ERR_INVALID_ARG; small or misaligned workspace -> ACE_ERR_WORKSPACE.
 */
/*
 * Offline per-expert amplification tables on the device: A^GSP by Alg. 2 (Eqs.
 * gsp_up_path, gsp_gate_path, gsp_geometric_mean, gsp_layer_normalization; the
 * Frobenius norms of the two [d, d] products come from m x m Gram matrices on fp64
 * MFMA) and A^RCR by Alg. 3 (Eqs. rcr_centered_router, rcr_direction_prototype with
 * rho = 1, rcr_raw_amplification with the prototype as the expert input,
 * rcr_layer_normalization).  fp64 throughout; deterministic.
 *   desc       reads N, d, m, dtype and eps (the other fields are ignored).
 *   w          reads gamma, w_router, w_gate, w_up, w_down (layouts as ace_moe_weights).
 *   a_gsp, a_rcr      DEVICE [N] fp32 out: the tables ace_moe_forward takes.
 *   a_gsp64, a_rcr64  DEVICE [N] fp64 out, optional (NULL).
 *   workspace  DEVICE scratch of ace_tables_workspace_size(desc) bytes, 256-byte aligned.
 * Requires m % 64 == 0 and d % 32 == 0 (else ACE_ERR_UNSUPPORTED).
 */
size_t ace_tables_workspace_size(const ace_moe_desc *desc);
ace_status ace_build_tables(const ace_moe_desc *desc, const ace_moe_weights *w, float *a_gsp, float *a_rcr,
                            double *a_gsp64, double *a_rcr64, void *workspace, size_t workspace_bytes,
                            void *stream);

#define ACE_TAU_MAX_Q 8
size_t ace_tau_workspace_size(void);
ace_status ace_tau_map(const float *scores, int64_t n_rows, int32_t k, int32_t m_min, const double *q,
                       int32_t n_q, float *tau, int64_t *m_q, int64_t *n_cand, void *workspace,
                       size_t workspace_bytes, void *stream);

/* Static, human-readable text of a status code (never NULL). */
const char *ace_status_string(int status);

/* ACE_ABI_VERSION of the built library. */
int ace_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ACE_H */
