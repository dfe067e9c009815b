"""Test-only fp64 numpy statement of the chunkwise gated delta rule.

This is neither the oracle nor the product: it writes out, one chunk at a
time and in plain numpy, the algebra that the HIP kernels implement, so that
the tests can check that algebra against the oracle's token recurrence at
several chunk sizes (including ragged last chunks).

State orientation: S is stored dk x dv (the transpose of the paper's
dv x dk state), so the paper's right-multiplied products become
left-multiplied.  Per chunk of n <= C tokens with entry state S
(Sec. 3.3, "Hardware-efficient chunkwise training"; Sec. 2.1 for the decay
notation, Eq. "def_notation"):

  g      = cumulative sum of log alpha inside the chunk (log of gamma^r)
  Gamma  = exp(g_r - g_i) for i <= r, else 0      (decay-aware causal mask)
  A      = strictLower(diag(beta) (Gamma * K K^T))
  T      = (I + A)^-1                              (gated UT transform)
  X      = diag(beta) (V - diag(e^g) K S)
  V'     = T X               (= U~ - W~ S with the paper's U~ and decayed W)
  O      = diag(e^g) Q S + (Gamma * Q K^T) V'
  S_next = e^{g_n} S + (diag(e^{g_n - g}) K)^T V'

Reading taken: the intra-chunk output mask is Gamma (with its diagonal), not
the plain causal mask M printed in the gated output equation; with M the
result disagrees with the recurrence (checked in the tests).

The backward is the exact reverse-mode derivative of those chunk equations
(the paper gives none); see ``chunk_bwd``.
"""
from __future__ import annotations

import numpy as np


def _chunk_tensors(Kc, Qc, bc, lc):
    g = np.cumsum(lc)
    n = len(lc)
    diff = g[:, None] - g[None, :]
    lower = np.tril(np.ones((n, n), dtype=bool))
    Gam = np.where(lower, np.exp(np.where(lower, diff, 0.0)), 0.0)  # select, never inf*0
    KK = Kc @ Kc.T
    Ak = np.tril(Gam * KK, -1)                    # strictLower(Gamma * K K^T), no beta
    A = bc[:, None] * Ak
    T = np.linalg.inv(np.eye(n) + A)
    P = Gam * (Qc @ Kc.T)                         # lower incl. diagonal
    return g, Gam, Ak, A, T, P


def chunk_fwd(q, k, v, beta, log_alpha, S0=None, C=64, output_mask="gamma"):
    """One (sequence, head): q,k [L,dk], v [L,dv], beta/log_alpha [L]."""
    L, dk = q.shape
    dv = v.shape[1]
    S = np.zeros((dk, dv)) if S0 is None else np.array(S0, dtype=np.float64)
    o = np.zeros((L, dv))
    for s in range(0, L, C):
        e = min(L, s + C)
        Qc, Kc, Vc, bc, lc = q[s:e], k[s:e], v[s:e], beta[s:e], log_alpha[s:e]
        g, Gam, Ak, A, T, P = _chunk_tensors(Kc, Qc, bc, lc)
        if output_mask == "M":  # the literal printed mask, kept only to show it is wrong
            P = np.tril(Qc @ Kc.T)
        eg = np.exp(g)
        X = bc[:, None] * (Vc - eg[:, None] * (Kc @ S))
        Vp = T @ X
        o[s:e] = eg[:, None] * (Qc @ S) + P @ Vp
        Kbar = np.exp(g[-1] - g)[:, None] * Kc
        S = np.exp(g[-1]) * S + Kbar.T @ Vp
    return o, S


def chunk_bwd(q, k, v, beta, log_alpha, dO, S0=None, dSf=None, C=64):
    """Reverse-mode derivative of ``chunk_fwd`` for one (sequence, head).

    Per chunk, with dS_next the gradient flowing into the chunk's exit state:
      dV'  = P^T dO + Kbar dS_next            dX = T^T dV'
      dS   = e^{g_n} dS_next + (diag(e^g) Q)^T dO - (diag(beta e^g) K)^T dX
      dV   = diag(beta) dX
      Gq = dO S^T,  Gk = dX S^T,  Gs = V' dS_next^T
      dP   = lower(dO V'^T),  dA = strictLower(-dX V'^T)
      dQ   = diag(e^g) Gq + (dP * Gamma) K
      D    = diag(beta) (dA * Gamma)
      dK   = (dP * Gamma)^T Q + diag(e^{g_n-g}) Gs - diag(beta e^g) Gk + (D + D^T) K
      dbeta_r = sum_i dA_ri Ak_ri + dX_r . V_r - e^{g_r} k_r . Gk_r
      E    = dA * diag(beta) Ak + dP * P
      dg_r = e^{g_r} q_r.Gq_r - beta_r e^{g_r} k_r.Gk_r - e^{g_n-g_r} k_r.Gs_r
             + sum_i E_ri - sum_j E_jr
      dg_last += sum_r e^{g_n-g_r} k_r.Gs_r + e^{g_n} <dS_next, S>
      dlog_alpha_j = sum_{r >= j in the chunk} dg_r
    """
    L, dk = q.shape
    dv = v.shape[1]
    S = np.zeros((dk, dv)) if S0 is None else np.array(S0, dtype=np.float64)
    starts = list(range(0, L, C))
    states = []
    for s in starts:  # forward, keeping the entry state of every chunk
        states.append(S.copy())
        e = min(L, s + C)
        Qc, Kc, Vc, bc, lc = q[s:e], k[s:e], v[s:e], beta[s:e], log_alpha[s:e]
        g, Gam, Ak, A, T, P = _chunk_tensors(Kc, Qc, bc, lc)
        eg = np.exp(g)
        X = bc[:, None] * (Vc - eg[:, None] * (Kc @ S))
        Vp = T @ X
        S = np.exp(g[-1]) * S + (np.exp(g[-1] - g)[:, None] * Kc).T @ Vp
    dq = np.zeros_like(q)
    dk_ = np.zeros_like(k)
    dv_ = np.zeros_like(v)
    db = np.zeros(L)
    dla = np.zeros(L)
    dS = np.zeros((dk, dv)) if dSf is None else np.array(dSf, dtype=np.float64)
    for ci in range(len(starts) - 1, -1, -1):
        s = starts[ci]
        e = min(L, s + C)
        S = states[ci]
        Qc, Kc, Vc, bc, lc, dOc = q[s:e], k[s:e], v[s:e], beta[s:e], log_alpha[s:e], dO[s:e]
        g, Gam, Ak, A, T, P = _chunk_tensors(Kc, Qc, bc, lc)
        eg = np.exp(g)
        egn = np.exp(g[-1])
        dec = np.exp(g[-1] - g)
        X = bc[:, None] * (Vc - eg[:, None] * (Kc @ S))
        Vp = T @ X
        dVp = P.T @ dOc + (dec[:, None] * Kc) @ dS
        dX = T.T @ dVp
        Gq = dOc @ S.T
        Gk = dX @ S.T
        Gs = Vp @ dS.T
        dP = np.tril(dOc @ Vp.T)
        dA = np.tril(-dX @ Vp.T, -1)
        M1 = dP * Gam
        D = bc[:, None] * (dA * Gam)
        dq[s:e] = eg[:, None] * Gq + M1 @ Kc
        dk_[s:e] = (M1.T @ Qc + dec[:, None] * Gs - (bc * eg)[:, None] * Gk + (D + D.T) @ Kc)
        dv_[s:e] = bc[:, None] * dX
        db[s:e] = (dA * Ak).sum(1) + (dX * Vc).sum(1) - eg * (Kc * Gk).sum(1)
        E = dA * (bc[:, None] * Ak) + dP * P
        ks = (Kc * Gs).sum(1)
        dg = (eg * (Qc * Gq).sum(1) - bc * eg * (Kc * Gk).sum(1) - dec * ks
              + E.sum(1) - E.sum(0))
        dg[-1] += (dec * ks).sum() + egn * (dS * S).sum()
        dla[s:e] = np.cumsum(dg[::-1])[::-1]
        dS = egn * dS + (eg[:, None] * Qc).T @ dOc - ((bc * eg)[:, None] * Kc).T @ dX
    return dict(dq=dq, dk=dk_, dv=dv_, dbeta=db, dlog_alpha=dla, dh0=dS)
