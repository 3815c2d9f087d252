"""Offline per-expert amplification tables in fp64 (test infrastructure only).

gsp_table  follows Alg. 2 (Global Spectral Proxy) with Eqs. gsp_up_path,
           gsp_gate_path, gsp_geometric_mean and gsp_layer_normalization (Sec. 3.1).
rcr_table  follows Alg. 3 (Router-Conditioned Refinement) with Eqs.
           rcr_centered_router, rcr_direction_prototype, rcr_raw_amplification and
           rcr_layer_normalization (Sec. 3.2).

Layouts are nn.Linear (out x in): w_gate/w_up [N, m, d], w_down [N, d, m].  The
paper writes row vectors times weights (x Gamma W), so its W^gate is w_gate^T
and Gamma scales the input (d) axis.  Frobenius norms are transpose invariant,
so || Gamma W^gate W^down ||_F = || w_down @ w_gate @ diag(gamma) ||_F.

The paper calls the proxy "spectral" but its equations and Alg. 2 use Frobenius
norms; the oracle uses Frobenius norms.
"""
from __future__ import annotations

import numpy as np

from .forward import expert_ffn, f64


def gsp_raw(gamma, w_gate_e, w_up_e, w_down_e):
    """Raw GSP amplification a~ of one expert (the per-expert body of Alg. 2)."""
    gam = f64(gamma)
    G = f64(w_gate_e) * gam[None, :]          # Gamma W^gate, as [m, d]
    U = f64(w_up_e) * gam[None, :]            # Gamma W^up
    Wd = f64(w_down_e)                        # [d, m]
    a_up = np.linalg.norm(U) * np.linalg.norm(Wd @ G)      # Eq. gsp_up_path
    a_gate = np.linalg.norm(G) * np.linalg.norm(Wd @ U)    # Eq. gsp_gate_path
    return np.sqrt(a_up * a_gate)                          # Eq. gsp_geometric_mean


def gsp_table(gamma, w_gate, w_up, w_down, eps: float = 1e-6):
    """A^GSP(e) = a~_e / (mean_j a~_j + eps) for every expert of one layer (Alg. 2)."""
    N = w_gate.shape[0]
    raw = np.array([gsp_raw(gamma, w_gate[e], w_up[e], w_down[e]) for e in range(N)])
    mu = raw.mean()
    return raw / (mu + eps)                                # Eq. gsp_layer_normalization


def rcr_prototypes(w_router, eps: float = 1e-6, rho: float = 1.0):
    """q_e = rho * w~_e / (RMS(w~_e) + eps), w~_e = w_e - mean_j w_j (Alg. 3)."""
    W = f64(w_router)
    w_bar = W.mean(axis=0)                                 # Eq. rcr_centered_router
    q = np.zeros_like(W)
    for e in range(W.shape[0]):
        wt = W[e] - w_bar
        r = np.sqrt(np.mean(wt * wt))
        q[e] = rho * wt / (r + eps)                        # Eq. rcr_direction_prototype
    return q


def rcr_raw(q_e, w_gate_e, w_up_e, w_down_e, eps: float = 1e-6, gamma=None):
    """a~^RCR = ||f_e(q_e)|| / (||q_e|| + eps)  (Eq. rcr_raw_amplification).

    f_e acts on q_e as the expert input x; with `gamma` given, the prototype is
    first scaled by Gamma (the alternative reading of where Gamma enters)."""
    x = f64(q_e) if gamma is None else f64(q_e) * f64(gamma)
    y = expert_ffn(x, w_gate_e, w_up_e, w_down_e)
    return np.linalg.norm(y) / (np.linalg.norm(f64(q_e)) + eps)


def rcr_table(w_router, w_gate, w_up, w_down, eps: float = 1e-6, rho: float = 1.0,
              gamma=None):
    """A^RCR(e) for every expert of one layer (Alg. 3)."""
    q = rcr_prototypes(w_router, eps, rho)
    N = q.shape[0]
    raw = np.array([rcr_raw(q[e], w_gate[e], w_up[e], w_down[e], eps, gamma) for e in range(N)])
    mu = raw.mean()
    return raw / (mu + eps)                                # Eq. rcr_layer_normalization


def build_tables(layer: dict, eps: float = 1e-6):
    """(A^GSP, A^RCR) of one layer in fp64 and their fp32 roundings (the values
    handed to both the GPU path and the oracle's online pass)."""
    a_gsp = gsp_table(layer["gamma"], layer["w_gate"], layer["w_up"], layer["w_down"], eps)
    a_rcr = rcr_table(layer["w_router"], layer["w_gate"], layer["w_up"], layer["w_down"], eps)
    return dict(a_gsp64=a_gsp, a_rcr64=a_rcr,
                a_gsp=a_gsp.astype(np.float32), a_rcr=a_rcr.astype(np.float32))
