"""Dense softmax attention in float64: the definition CQS decomposition
reproduces exactly.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Layout: Q, K, V, dO are [B, L, H, d] arrays holding the *stored* input values
(16-bit or fp32 inputs are converted exactly to float64).  The softmax scale
is alpha = 1/sqrt(d) unless given (Section 3.1, below Eq. 2).  Causal
attention keeps key j for query i iff j <= i, in global token order.

Forward (Section 3.1, Eqs. 2-3 read without decomposition, i.e. one task
holding all tokens and an all-ones mask):
    S = alpha * Q K^T,   P = softmax_rows(S),   O = P V,
    LSE = m + ln(sum_j exp(S_j - m)),   m = max_j S_j   (App. A.1, below
    Eq. "merge": lse = m + log l).

Backward (App. A.1, Eq. "globallse", which the paper shows equal to Alg. 2 /
App. D): with P[q,k] = exp(S[q,k] - LSE[q]) and D[q] = sum_d dO[q]*O[q],
    dV = P^T dO,  dP = dO V^T,  dS = P * (dP - D),
    dQ = alpha dS K,  dK = alpha dS^T Q.
"""
import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _scale(d, scale):
    return 1.0 / np.sqrt(d) if scale is None else float(scale)


def attention_forward(Q, K, V, causal, scale=None, rows=None, row_chunk=16):
    """Dense forward on a subset of query rows.

    Q, K, V: [B, L, H, d].  rows: None (all rows) or an int array of query
    indices, shared by every (b, h), or a list of H such arrays (one per head).
    Returns O [B, R, H, d] (or a list per head when rows is per head) and
    LSE [B, H, R], both float64.  Rows are processed row_chunk at a time so a
    1M-key row set needs only row_chunk * L * 8 bytes of scores.
    """
    Q = np.asarray(Q)
    B, L, H, d = Q.shape
    alpha = _scale(d, scale)
    per_head = isinstance(rows, (list, tuple))
    if rows is None:
        rows_h = [np.arange(L)] * H
    elif per_head:
        rows_h = [np.asarray(r, dtype=np.int64) for r in rows]
    else:
        rows_h = [np.asarray(rows, dtype=np.int64)] * H
    R = len(rows_h[0])
    O = np.zeros((B, R, H, d))
    LSE = np.zeros((B, H, R))
    for b in range(B):
        for h in range(H):
            k = _f64(K[b, :, h, :])
            v = _f64(V[b, :, h, :])
            r_all = rows_h[h]
            for c0 in range(0, R, row_chunk):
                r = r_all[c0:c0 + row_chunk]
                q = _f64(Q[b, r, h, :])
                s = alpha * (q @ k.T)                       # [r, L]
                if causal:
                    keep = np.arange(L)[None, :] <= r[:, None]
                    s = np.where(keep, s, -np.inf)
                m = s.max(axis=1, keepdims=True)
                p = np.exp(s - m)
                denom = p.sum(axis=1, keepdims=True)
                O[b, c0:c0 + len(r), h, :] = (p @ v) / denom
                LSE[b, h, c0:c0 + len(r)] = (m + np.log(denom))[:, 0]
    return O, LSE


def attention_backward(Q, K, V, dO, causal, scale=None):
    """Dense analytic gradients on all rows (small L only: O(L^2) memory).

    Returns (dQ, dK, dV, O, LSE) in float64 with the input layouts.
    """
    Q = _f64(Q); K = _f64(K); V = _f64(V); dO = _f64(dO)
    B, L, H, d = Q.shape
    alpha = _scale(d, scale)
    dQ = np.zeros_like(Q); dK = np.zeros_like(K); dV = np.zeros_like(V)
    O = np.zeros_like(Q); LSE = np.zeros((B, H, L))
    keep = np.tril(np.ones((L, L), dtype=bool)) if causal else np.ones((L, L), dtype=bool)
    for b in range(B):
        for h in range(H):
            q = Q[b, :, h, :]; k = K[b, :, h, :]; v = V[b, :, h, :]; do = dO[b, :, h, :]
            s = np.where(keep, alpha * (q @ k.T), -np.inf)
            m = s.max(axis=1, keepdims=True)
            lse = m + np.log(np.exp(s - m).sum(axis=1, keepdims=True))
            p = np.exp(s - lse)                              # rows sum to 1
            o = p @ v
            D = (do * o).sum(axis=1, keepdims=True)
            dp = do @ v.T
            ds = p * (dp - D)
            dQ[b, :, h, :] = alpha * (ds @ k)
            dK[b, :, h, :] = alpha * (ds.T @ q)
            dV[b, :, h, :] = p.T @ do
            O[b, :, h, :] = o
            LSE[b, h, :] = lse[:, 0]
    return dQ, dK, dV, O, LSE


def attention_backward_rows(Q, K, V, dO, causal, q_rows, k_rows, scale=None, row_chunk=64):
    """The gradients of `attention_backward` on a subset of rows, for long
    sequences: dQ on query rows q_rows and dK, dV on key rows k_rows.

    Same definitions (App. A.1, Eq. "globallse").  A dQ row needs only its own
    query's scores; a dK or dV row sums over every query that keeps the key,
    so every query row is visited once, row_chunk at a time: its scores give
    its LSE, P row, O row and D, and its contribution to the sampled keys'
    sums is added before the next chunk.  Memory is row_chunk * L scores;
    time is O(L^2 d) per (b, h).

    q_rows, k_rows: int arrays shared by every head, or lists of H arrays.
    Returns dQ [B, len(q_rows), H, d] and dK, dV [B, len(k_rows), H, d], float64.
    """
    Q = np.asarray(Q)
    B, L, H, d = Q.shape
    alpha = _scale(d, scale)
    per_head = lambda r: ([np.asarray(x, dtype=np.int64) for x in r]
                          if isinstance(r, (list, tuple)) else [np.asarray(r, dtype=np.int64)] * H)
    qr_h, kr_h = per_head(q_rows), per_head(k_rows)
    dQ = np.zeros((B, len(qr_h[0]), H, d))
    dK = np.zeros((B, len(kr_h[0]), H, d))
    dV = np.zeros((B, len(kr_h[0]), H, d))
    for b in range(B):
        for h in range(H):
            k = _f64(K[b, :, h, :]); v = _f64(V[b, :, h, :])
            kr = kr_h[h]
            qpos = {int(r): i for i, r in enumerate(qr_h[h])}
            for c0 in range(0, L, row_chunk):
                r = np.arange(c0, min(L, c0 + row_chunk))
                q = _f64(Q[b, r, h, :]); do = _f64(dO[b, r, h, :])
                s = alpha * (q @ k.T)                                  # [r, L]
                if causal:
                    s = np.where(np.arange(L)[None, :] <= r[:, None], s, -np.inf)
                m = s.max(axis=1, keepdims=True)
                lse = m + np.log(np.exp(s - m).sum(axis=1, keepdims=True))
                p = np.exp(s - lse)                                    # rows sum to 1
                D = (do * (p @ v)).sum(axis=1, keepdims=True)
                # the sampled keys' columns of dS for these queries
                ds_k = p[:, kr] * (do @ v[kr].T - D)
                dK[b, :, h, :] += alpha * (ds_k.T @ q)
                dV[b, :, h, :] += p[:, kr].T @ do
                sel = [i for i, x in enumerate(r) if int(x) in qpos]
                if sel:
                    ds = p[sel] * (do[sel] @ v.T - D[sel])
                    dQ[b, [qpos[int(r[i])] for i in sel], h, :] = alpha * (ds @ k)
    return dQ, dK, dV


def rel_l2(x, ref):
    """Relative error ||x - ref||_2 / ||ref||_2 over the whole tensor, the
    metric read into Section 4.2's "relative error"."""
    x = _f64(x); ref = _f64(ref)
    return float(np.linalg.norm((x - ref).ravel()) / np.linalg.norm(ref.ravel()))
