// Offline per-expert amplification tables on the device, in fp64:
//   GSP (Alg. 2): with G = W_gate diag(gamma), U = W_up diag(gamma) ([m, d],
//     nn.Linear layout) and W_down [d, m],
//       a_up = ||U||_F ||W_down G||_F, a_gate = ||G||_F ||W_down U||_F
//       (Eqs. gsp_up_path, gsp_gate_path), a~ = sqrt(a_up a_gate)
//       (Eq. gsp_geometric_mean), A = a~ / (mean a~ + eps) (Eq. gsp_layer_normalization).
//     The two [d, d] products are never formed: ||W_down G||_F^2 =
//     <W_down^T W_down, G G^T>_F, an inner product of two m x m Gram matrices
//     (about 1.8x fewer flops than the products).  gsp_tile_kernel computes,
//     per expert and per 64 x 64 tile pair (bi <= bj) of the m x m space, the
//     tiles of W_down^T W_down, G G^T and U U^T on fp64 MFMA
//     (v_mfma_f64_16x16x4f64) and reduces sum(D o G) and sum(D o U) over the
//     tile; the Gram matrices are symmetric, so an off-diagonal pair counts
//     twice.
//   RCR (Alg. 3): w~_e = w_e - mean_j w_j (Eq. rcr_centered_router),
//     q_e = rho w~_e / (RMS(w~_e) + eps) with rho = 1 (Eq. rcr_direction_prototype),
//     a~ = ||f_e(q_e)|| / (||q_e|| + eps) with f_e the SwiGLU expert applied to
//     q_e as its input (Eq. rcr_raw_amplification), A = a~ / (mean a~ + eps)
//     (Eq. rcr_layer_normalization).  One workgroup per expert, fp64 VALU
//     (about 3 m d multiply-adds per expert).  The same pass accumulates
//     ||G||_F^2 and ||U||_F^2 for GSP.
// Every reduction has a fixed order, so the tables are deterministic; fp64
// throughout, they agree with an fp64 evaluation to ~1e-15 relative.
#include "ace_internal.h"

namespace ace {

namespace {

typedef double f64x4_t __attribute__((ext_vector_type(4)));

// 8 consecutive elements as raw storage; element i as a double
template <typename T> struct Raw8;
template <> struct Raw8<bf16_t> {
  uint4 v;
  __device__ __forceinline__ void load(const bf16_t *p) { v = *reinterpret_cast<const uint4 *>(p); }
  __device__ __forceinline__ double at(int i) const {
    const uint32_t w = i < 2 ? v.x : i < 4 ? v.y : i < 6 ? v.z : v.w;
    return static_cast<double>(__uint_as_float((i & 1) ? (w & 0xFFFF0000u) : (w << 16)));
  }
};
template <> struct Raw8<float> {
  float4 lo, hi;
  __device__ __forceinline__ void load(const float *p) {
    lo = *reinterpret_cast<const float4 *>(p);
    hi = *reinterpret_cast<const float4 *>(p + 4);
  }
  __device__ __forceinline__ double at(int i) const {
    const float4 &h = i < 4 ? lo : hi;
    const int j = i & 3;
    return static_cast<double>(j == 0 ? h.x : j == 1 ? h.y : j == 2 ? h.z : h.w);
  }
};

__device__ __forceinline__ double to_f64(bf16_t v) { return static_cast<double>(bf16_to_f32(v)); }
__device__ __forceinline__ double to_f64(float v) { return static_cast<double>(v); }

struct TabArgs {
  const void *gamma, *w_router, *w_gate, *w_up, *w_down;
  int N, d, m, mt, n_pairs;
  double eps, rho;
  double *pair_part;  // [N][n_pairs][2]: sum(D o G), sum(D o U) of each tile pair
  double *wbar;       // [d] mean router row
  double *rcr_raw;    // [N]
  double *norm2;      // [N][2]: ||G||_F^2, ||U||_F^2
  double *gsp_raw;    // [N]
  float *a_gsp, *a_rcr;
  double *a_gsp64, *a_rcr64;
};

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// grid (tile pairs, experts), 4 waves; wave (wr, wc) owns a 32 x 32 sub-tile
template <typename T>
__global__ __launch_bounds__(256) void gsp_tile_kernel(TabArgs a) {
  const int e = blockIdx.y;
  int p = blockIdx.x, bi = 0;
  while (p >= a.mt - bi) {
    p -= a.mt - bi;
    ++bi;
  }
  const int bj = bi + p;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int wr = wave >> 1, wc = wave & 1;
  const int d = a.d, m = a.m;
  const size_t eo = static_cast<size_t>(e) * m * d;
  const T *Wg = static_cast<const T *>(a.w_gate) + eo;
  const T *Wu = static_cast<const T *>(a.w_up) + eo;
  const T *Wd = static_cast<const T *>(a.w_down) + eo;  // [d, m]
  const T *gam = static_cast<const T *>(a.gamma);
  int ri[2], cj[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    ri[u] = bi * 64 + wr * 32 + 16 * u + r16;
    cj[u] = bj * 64 + wc * 32 + 16 * u + r16;
  }
  f64x4_t accD[2][2], accG[2][2], accU[2][2];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v) accD[u][v] = accG[u][v] = accU[u][v] = f64x4_t{0.0, 0.0, 0.0, 0.0};

  // 32-wide K blocks; lane group g holds k = k0 + 8 g + j and MFMA j takes element j
  for (int k0 = 0; k0 < d; k0 += 32) {
    const int kb = k0 + 8 * g;
    Raw8<T> gm, ga[2], gb[2], ua[2], ub[2];
    gm.load(gam + kb);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      ga[u].load(Wg + static_cast<size_t>(ri[u]) * d + kb);
      gb[u].load(Wg + static_cast<size_t>(cj[u]) * d + kb);
      ua[u].load(Wu + static_cast<size_t>(ri[u]) * d + kb);
      ub[u].load(Wu + static_cast<size_t>(cj[u]) * d + kb);
    }
    T da[2][8], db[2][8];  // W_down[k][col] for the 8 k of this lane group
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        da[u][j] = Wd[static_cast<size_t>(kb + j) * m + ri[u]];
        db[u][j] = Wd[static_cast<size_t>(kb + j) * m + cj[u]];
      }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const double gj = gm.at(j);
      double xa[2], xb[2], ya[2], yb[2], za[2], zb[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        xa[u] = ga[u].at(j) * gj;
        xb[u] = gb[u].at(j) * gj;
        ya[u] = ua[u].at(j) * gj;
        yb[u] = ub[u].at(j) * gj;
        za[u] = to_f64(da[u][j]);
        zb[u] = to_f64(db[u][j]);
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int v = 0; v < 2; ++v) {
          accG[u][v] = __builtin_amdgcn_mfma_f64_16x16x4f64(xa[u], xb[v], accG[u][v], 0, 0, 0);
          accU[u][v] = __builtin_amdgcn_mfma_f64_16x16x4f64(ya[u], yb[v], accU[u][v], 0, 0, 0);
          accD[u][v] = __builtin_amdgcn_mfma_f64_16x16x4f64(za[u], zb[v], accD[u][v], 0, 0, 0);
        }
    }
  }
  // sum(D o G), sum(D o U) over this wave's sub-tile (the three tiles share one layout)
  double sg = 0.0, su = 0.0;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sg = fma(accD[u][v][i], accG[u][v][i], sg);
        su = fma(accD[u][v][i], accU[u][v][i], su);
      }
  sg = wave_sum(sg);
  su = wave_sum(su);
  __shared__ double part[4][2];
  if (lane == 0) {
    part[wave][0] = sg;
    part[wave][1] = su;
  }
  __syncthreads();
  if (tid == 0) {
    const double mult = bi == bj ? 1.0 : 2.0;
    double tg = 0.0, tu = 0.0;
    for (int w = 0; w < 4; ++w) {
      tg += part[w][0];
      tu += part[w][1];
    }
    double *o = a.pair_part + (static_cast<size_t>(e) * a.n_pairs + blockIdx.x) * 2;
    o[0] = mult * tg;
    o[1] = mult * tu;
  }
}

// mean router row, one thread per column, experts added in order
template <typename T>
__global__ __launch_bounds__(256) void rcr_mean_kernel(TabArgs a) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= a.d) return;
  const T *W = static_cast<const T *>(a.w_router);
  double s = 0.0;
  for (int e = 0; e < a.N; ++e) s += to_f64(W[static_cast<size_t>(e) * a.d + k]);
  a.wbar[k] = s / a.N;
}

// block-wide sum in a fixed order (wave butterflies, then waves in order)
__device__ __forceinline__ double block_sum4(double v, double *scratch) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  return ((scratch[0] + scratch[1]) + scratch[2]) + scratch[3];
}

// one workgroup (4 waves) per expert
template <typename T>
__global__ __launch_bounds__(256) void rcr_expert_kernel(TabArgs a) {
  extern __shared__ double h[];  // [m]
  __shared__ double red[4];
  __shared__ double nrm[4][2];
  const int e = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = a.d, m = a.m;
  const T *wr = static_cast<const T *>(a.w_router) + static_cast<size_t>(e) * d;
  const T *gam = static_cast<const T *>(a.gamma);
  // RMS of the centred router row and ||q||
  double s2 = 0.0;
  for (int k = tid; k < d; k += 256) {
    const double w = to_f64(wr[k]) - a.wbar[k];
    s2 += w * w;
  }
  const double r = sqrt(block_sum4(s2, red) / d);
  const double inv = a.rho / (r + a.eps);
  double q2 = 0.0;
  for (int k = tid; k < d; k += 256) {
    const double q = (to_f64(wr[k]) - a.wbar[k]) * inv;
    q2 += q * q;
  }
  const double qn = sqrt(block_sum4(q2, red));
  // h = SiLU(W_gate q) * (W_up q); wave w takes rows w, w + 4, ...; also ||G||^2, ||U||^2
  const size_t eo = static_cast<size_t>(e) * m * d;
  const T *Wg = static_cast<const T *>(a.w_gate) + eo;
  const T *Wu = static_cast<const T *>(a.w_up) + eo;
  double ng = 0.0, nu = 0.0;
  for (int i = wave; i < m; i += 4) {
    double sgi = 0.0, sui = 0.0;
    for (int k = lane; k < d; k += 64) {
      const double q = (to_f64(wr[k]) - a.wbar[k]) * inv;
      const double wg = to_f64(Wg[static_cast<size_t>(i) * d + k]);
      const double wu = to_f64(Wu[static_cast<size_t>(i) * d + k]);
      sgi = fma(wg, q, sgi);
      sui = fma(wu, q, sui);
      const double gk = to_f64(gam[k]);
      const double G = wg * gk, U = wu * gk;
      ng = fma(G, G, ng);
      nu = fma(U, U, nu);
    }
    sgi = wave_sum(sgi);
    sui = wave_sum(sui);
    if (lane == 0) h[i] = sgi / (1.0 + exp(-sgi)) * sui;
  }
  ng = wave_sum(ng);
  nu = wave_sum(nu);
  if (lane == 0) {
    nrm[wave][0] = ng;
    nrm[wave][1] = nu;
  }
  __syncthreads();
  // f = W_down h; wave w takes rows w, w + 4, ...
  const T *Wd = static_cast<const T *>(a.w_down) + eo;
  double f2 = 0.0;
  for (int rr = wave; rr < d; rr += 4) {
    double s = 0.0;
    for (int i = lane; i < m; i += 64) s = fma(to_f64(Wd[static_cast<size_t>(rr) * m + i]), h[i], s);
    s = wave_sum(s);
    f2 = fma(s, s, f2);  // identical in every lane of the wave
  }
  if (lane == 0) red[wave] = f2;
  __syncthreads();
  if (tid == 0) {
    const double fn = sqrt(((red[0] + red[1]) + red[2]) + red[3]);
    a.rcr_raw[e] = fn / (qn + a.eps);
    a.norm2[2 * e] = ((nrm[0][0] + nrm[1][0]) + nrm[2][0]) + nrm[3][0];
    a.norm2[2 * e + 1] = ((nrm[0][1] + nrm[1][1]) + nrm[2][1]) + nrm[3][1];
  }
}

// GSP raw values from the tile sums, then both layer normalisations
__global__ __launch_bounds__(256) void tables_finalize_kernel(TabArgs a) {
  __shared__ double red[4];
  const int tid = threadIdx.x;
  double sg_all = 0.0, sr_all = 0.0;
  for (int e = tid; e < a.N; e += 256) {
    const double *pp = a.pair_part + static_cast<size_t>(e) * a.n_pairs * 2;
    double dg = 0.0, du = 0.0;
    for (int p = 0; p < a.n_pairs; ++p) {
      dg += pp[2 * p];
      du += pp[2 * p + 1];
    }
    const double a_up = sqrt(a.norm2[2 * e + 1]) * sqrt(dg);    // ||U|| ||W_d G||
    const double a_gate = sqrt(a.norm2[2 * e]) * sqrt(du);      // ||G|| ||W_d U||
    const double raw = sqrt(a_up * a_gate);
    a.gsp_raw[e] = raw;
    sg_all += raw;
    sr_all += a.rcr_raw[e];
  }
  const double mg = block_sum4(sg_all, red) / a.N;
  const double mr = block_sum4(sr_all, red) / a.N;
  for (int e = tid; e < a.N; e += 256) {
    const double ag = a.gsp_raw[e] / (mg + a.eps);
    const double ar = a.rcr_raw[e] / (mr + a.eps);
    a.a_gsp[e] = static_cast<float>(ag);
    a.a_rcr[e] = static_cast<float>(ar);
    if (a.a_gsp64) a.a_gsp64[e] = ag;
    if (a.a_rcr64) a.a_rcr64[e] = ar;
  }
}

template <typename T>
void launch_tables_t(const TabArgs &a, hipStream_t stream) {
  gsp_tile_kernel<T><<<dim3(a.n_pairs, a.N), 256, 0, stream>>>(a);
  rcr_mean_kernel<T><<<dim3((a.d + 255) / 256), 256, 0, stream>>>(a);
  rcr_expert_kernel<T><<<dim3(a.N), 256, static_cast<size_t>(a.m) * sizeof(double), stream>>>(a);
  tables_finalize_kernel<<<1, 256, 0, stream>>>(a);
}

size_t al(size_t v) { return (v + 255) / 256 * 256; }

}  // namespace

size_t tables_workspace_bytes(int N, int d, int m) {
  const size_t mt = static_cast<size_t>(m) / 64, np = mt * (mt + 1) / 2;
  return al(static_cast<size_t>(N) * np * 2 * 8) + al(static_cast<size_t>(d) * 8) + 3 * al(static_cast<size_t>(N) * 2 * 8);
}

hipError_t launch_tables(const TablesCall &c, hipStream_t stream) {
  TabArgs a{};
  a.gamma = c.gamma;
  a.w_router = c.w_router;
  a.w_gate = c.w_gate;
  a.w_up = c.w_up;
  a.w_down = c.w_down;
  a.N = c.N;
  a.d = c.d;
  a.m = c.m;
  a.mt = c.m / 64;
  a.n_pairs = a.mt * (a.mt + 1) / 2;
  a.eps = c.eps;
  a.rho = 1.0;
  char *ws = static_cast<char *>(c.workspace);
  a.pair_part = reinterpret_cast<double *>(ws);
  ws += al(static_cast<size_t>(c.N) * a.n_pairs * 2 * 8);
  a.wbar = reinterpret_cast<double *>(ws);
  ws += al(static_cast<size_t>(c.d) * 8);
  a.rcr_raw = reinterpret_cast<double *>(ws);
  ws += al(static_cast<size_t>(c.N) * 2 * 8);
  a.norm2 = reinterpret_cast<double *>(ws);
  ws += al(static_cast<size_t>(c.N) * 2 * 8);
  a.gsp_raw = reinterpret_cast<double *>(ws);
  a.a_gsp = c.a_gsp;
  a.a_rcr = c.a_rcr;
  a.a_gsp64 = c.a_gsp64;
  a.a_rcr64 = c.a_rcr64;
  if (c.bf16)
    launch_tables_t<bf16_t>(a, stream);
  else
    launch_tables_t<float>(a, stream);
  return hipGetLastError();
}

}  // namespace ace
