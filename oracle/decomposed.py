"""Decomposed attention in float64: forward and backward over CQS tasks.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Tasks come from ``oracle.planner.build_tasks``; Q, K, V, dO are [B, L, H, d]
arrays.  Every function here must equal ``oracle.dense`` up to float64
rounding, which the tests check by brute force.

* ``numden_forward`` / ``numden_backward``: Alg. 1 and Alg. 2 (Section 3.1,
  Eqs. 2-3; Section 3.2, Eqs. 4-6; App. D) written out literally:
  P_i = exp(R_i) * M_i with no max shift.  They overflow once
  lse > ln(FLT_MAX) in float32 (App. A.1), which is why the paper replaces
  them with the two functions below; in float64 they are exact for moderate
  scores and serve as a second derivation of the same result.
* ``merged_forward``: each task returns (acc_i, l_i, m_i); a global
  (acc, l, m) absorbs them with the max-shifted merge of App. A.1, Eq.
  "merge"; O = acc / l and lse = m + log l.  A task row with no kept key has
  m_i = -inf and is skipped as a null contribution (App. A.1, last paragraph
  of "Statistics in fp32").
* ``globallse_backward``: App. A.1, Eq. "globallse": every task recomputes
  P = exp(S - lse_global) on the pairs it keeps, runs the standard softmax
  backward with D = rowsum(dO * O), and its gradients are scatter-added.
"""
import numpy as np

from .planner import local_mask


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _alpha(d, scale):
    return 1.0 / np.sqrt(d) if scale is None else float(scale)


def task_statistics(Q, K, V, task, causal, scale=None):
    """Local statistics of one task: acc_i [B, Li, H, d], l_i [B, H, Li],
    m_i [B, H, Li] (natural-log domain), with null rows (m_i = -inf,
    l_i = 0, acc_i = 0)."""
    B, L, H, d = np.shape(Q)
    alpha = _alpha(d, scale)
    g = task["tokens"]
    keep = local_mask(task, causal)
    Li = len(g)
    acc = np.zeros((B, Li, H, d)); ell = np.zeros((B, H, Li)); m = np.full((B, H, Li), -np.inf)
    for b in range(B):
        for h in range(H):
            q = _f64(Q[b, g, h, :]); k = _f64(K[b, g, h, :]); v = _f64(V[b, g, h, :])
            s = np.where(keep, alpha * (q @ k.T), -np.inf)
            mm = s.max(axis=1) if Li else np.zeros(0)
            live = np.isfinite(mm)
            p = np.zeros_like(s)
            p[live] = np.exp(s[live] - mm[live][:, None])
            acc[b, :, h, :] = p @ v
            ell[b, h, :] = p.sum(axis=1)
            m[b, h, :] = np.where(live, mm, -np.inf)
    return acc, ell, m


def merge_into(acc, ell, m, task_tokens, acc_i, ell_i, m_i):
    """Eq. "merge" at the task's global rows, in place; skips null rows."""
    for b in range(acc.shape[0]):
        for h in range(acc.shape[2]):
            for r, gq in enumerate(task_tokens):
                mi = m_i[b, h, r]
                if not np.isfinite(mi):
                    continue                      # null contribution
                mo = m[b, h, gq]
                mn = max(mo, mi)
                a_old = np.exp(mo - mn) if np.isfinite(mo) else 0.0
                a_new = np.exp(mi - mn)
                acc[b, gq, h, :] = acc[b, gq, h, :] * a_old + acc_i[b, r, h, :] * a_new
                ell[b, h, gq] = ell[b, h, gq] * a_old + ell_i[b, h, r] * a_new
                m[b, h, gq] = mn


def merged_forward(Q, K, V, tasks, causal, scale=None, order=None):
    """Decomposed forward with the max-shifted merge.  `order` permutes the
    task sequence (the merge is order independent).  Returns O [B, L, H, d]
    and LSE [B, H, L]."""
    B, L, H, d = np.shape(Q)
    acc = np.zeros((B, L, H, d)); ell = np.zeros((B, H, L)); m = np.full((B, H, L), -np.inf)
    idx = range(len(tasks)) if order is None else order
    for t in idx:
        task = tasks[t]
        acc_i, ell_i, m_i = task_statistics(Q, K, V, task, causal, scale)
        merge_into(acc, ell, m, task["tokens"], acc_i, ell_i, m_i)
    O = acc / ell.transpose(0, 2, 1)[..., None]
    LSE = m + np.log(ell)
    return O, LSE


def numden_forward(Q, K, V, tasks, causal, scale=None, dtype=np.float64):
    """Alg. 1 literally (Num/Den, no max shift) in `dtype`.  Returns O, Num, Den."""
    B, L, H, d = np.shape(Q)
    alpha = dtype(_alpha(d, scale))
    Num = np.zeros((B, H, L, d), dtype=dtype); Den = np.zeros((B, H, L), dtype=dtype)
    with np.errstate(over="ignore", invalid="ignore"):
        for task in tasks:
            g = task["tokens"]
            M = local_mask(task, causal).astype(dtype)
            for b in range(B):
                for h in range(H):
                    q = np.asarray(Q[b, g, h, :], dtype=dtype)
                    k = np.asarray(K[b, g, h, :], dtype=dtype)
                    v = np.asarray(V[b, g, h, :], dtype=dtype)
                    R = alpha * (q @ k.T)
                    P = np.exp(R) * M
                    np.add.at(Num[b, h], g, P @ v)
                    np.add.at(Den[b, h], g, P.sum(axis=1))
        O = Num / Den[..., None]
    return O.transpose(0, 2, 1, 3), Num, Den


def numden_backward(Q, K, V, dO, tasks, causal, scale=None):
    """Alg. 2 literally in float64 (dNum = dO/Den, dDen = -<dO,Num>/Den^2,
    per task dV_i, dP_i, dR_i, dQ_i, dK_i, scatter-added)."""
    B, L, H, d = np.shape(Q)
    alpha = _alpha(d, scale)
    _, Num, Den = numden_forward(Q, K, V, tasks, causal, scale)
    dOt = _f64(dO).transpose(0, 2, 1, 3)                       # [B, H, L, d]
    dNum = dOt / Den[..., None]
    dDen = -(dOt * Num).sum(axis=-1) / (Den * Den)
    dQ = np.zeros((B, H, L, d)); dK = np.zeros((B, H, L, d)); dV = np.zeros((B, H, L, d))
    for task in tasks:
        g = task["tokens"]
        M = local_mask(task, causal).astype(np.float64)
        for b in range(B):
            for h in range(H):
                q = _f64(Q[b, g, h, :]); k = _f64(K[b, g, h, :]); v = _f64(V[b, g, h, :])
                P = np.exp(alpha * (q @ k.T)) * M
                dn = dNum[b, h, g]; dd = dDen[b, h, g]
                dVi = P.T @ dn
                dPi = dn @ v.T + dd[:, None]
                dRi = dPi * P
                np.add.at(dQ[b, h], g, alpha * (dRi @ k))
                np.add.at(dK[b, h], g, alpha * (dRi.T @ q))
                np.add.at(dV[b, h], g, dVi)
    tr = lambda x: x.transpose(0, 2, 1, 3)
    return tr(dQ), tr(dK), tr(dV)


def globallse_backward(Q, K, V, dO, O, LSE, tasks, causal, scale=None):
    """Eq. "globallse" backward: per task P = exp(S - LSE[q]) * M_i,
    D = rowsum(dO * O), dS = P * (dP - D); gradients scatter-added."""
    B, L, H, d = np.shape(Q)
    alpha = _alpha(d, scale)
    D = (_f64(dO) * _f64(O)).sum(axis=-1)                      # [B, L, H]
    dQ = np.zeros((B, L, H, d)); dK = np.zeros((B, L, H, d)); dV = np.zeros((B, L, H, d))
    for task in tasks:
        g = task["tokens"]
        keep = local_mask(task, causal)
        for b in range(B):
            for h in range(H):
                q = _f64(Q[b, g, h, :]); k = _f64(K[b, g, h, :]); v = _f64(V[b, g, h, :])
                do = _f64(dO[b, g, h, :])
                s = alpha * (q @ k.T)
                P = np.where(keep, np.exp(np.where(keep, s, 0.0) - _f64(LSE[b, h, g])[:, None]), 0.0)
                dp = do @ v.T
                ds = P * (dp - D[b, g, h][:, None])
                np.add.at(dQ[b, :, h, :], g, alpha * (ds @ k))
                np.add.at(dK[b, :, h, :], g, alpha * (ds.T @ q))
                np.add.at(dV[b, :, h, :], g, P.T @ do)
    return dQ, dK, dV


def row_mass(Q, K, tasks, LSE, causal, scale=None):
    """Sum over tasks of sum over kept keys of exp(S - LSE): the softmax row
    mass recovered from the pieces, which must be 1 for every row."""
    B, L, H, d = np.shape(Q)
    alpha = _alpha(d, scale)
    mass = np.zeros((B, H, L))
    for task in tasks:
        g = task["tokens"]
        keep = local_mask(task, causal)
        for b in range(B):
            for h in range(H):
                q = _f64(Q[b, g, h, :]); k = _f64(K[b, g, h, :])
                s = alpha * (q @ k.T)
                P = np.where(keep, np.exp(np.where(keep, s, 0.0) - _f64(LSE[b, h, g])[:, None]), 0.0)
                np.add.at(mass[b, h], g, P.sum(axis=1))
    return mass
