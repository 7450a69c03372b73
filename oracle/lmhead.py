"""Oracle: LM-head log-probabilities and their backward
(test infrastructure only; see oracle/__init__).

Paper, Sec. 3.2 (post-pruning evaluation): the kept trajectories' hidden states are
projected through the output layer to logits, a softmax over the vocabulary gives
token probabilities, and the sampled token's probability enters the ratios.  Here:

    z[t, v]  = sum_k H[t, k] * W[v, k]                      (logits)
    lse[t]   = m_t + log sum_v exp(z[t, v] - m_t),  m_t = max_v z[t, v]
    logp[t]  = z[t, y_t] - lse[t]

Backward of a loss L whose derivative w.r.t. logp[t] is g[t] (Sec. 3.1: the gradient
is a weighted sum of grad log pi over tokens):

    dZ[t, v] = g[t] * (1[v == y_t] - exp(z[t, v] - lse[t]))
    dH       = dZ @ W,      dW = dZ^T @ H

Policy entropy per token (the statistic the paper follows during training, Sec. 4,
entropy curves), from its definition over the softmax:

    H[t] = - sum_v p[t, v] log p[t, v],    p[t, v] = exp(z[t, v] - lse[t])

All arithmetic is float64; rows are processed in chunks only to bound memory (rows
are independent, so chunking changes nothing but the summation order of dW).
"""
import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def logits(H, W):
    return _f64(H) @ _f64(W).T


def token_logprob(H, W, y, row_chunk=64):
    """Return (logp float64[T], lse float64[T])."""
    H = _f64(H)
    W = _f64(W)
    y = np.asarray(y, dtype=np.int64)
    T = H.shape[0]
    logp = np.empty(T, dtype=np.float64)
    lse = np.empty(T, dtype=np.float64)
    for a in range(0, T, row_chunk):
        b = min(T, a + row_chunk)
        z = H[a:b] @ W.T
        m = z.max(axis=1)
        s = np.exp(z - m[:, None]).sum(axis=1)
        l = m + np.log(s)
        lse[a:b] = l
        logp[a:b] = z[np.arange(b - a), y[a:b]] - l
    return logp, lse


def lmhead_backward(H, W, y, lse, g, row_chunk=64, need_dW=True):
    """Return (dH float64[T, d], dW float64[V, d] or None)."""
    H = _f64(H)
    W = _f64(W)
    y = np.asarray(y, dtype=np.int64)
    lse = _f64(lse)
    g = _f64(g)
    T, d = H.shape
    V = W.shape[0]
    dH = np.empty((T, d), dtype=np.float64)
    dW = np.zeros((V, d), dtype=np.float64) if need_dW else None
    for a in range(0, T, row_chunk):
        b = min(T, a + row_chunk)
        z = H[a:b] @ W.T
        dz = -np.exp(z - lse[a:b, None])
        dz[np.arange(b - a), y[a:b]] += 1.0
        dz *= g[a:b, None]
        dH[a:b] = dz @ W
        if need_dW:
            dW += dz.T @ H[a:b]
    return dH, dW


def lmhead_dW_rows(H, W, y, lse, g, vocab_rows, row_chunk=4096):
    """Exact dW rows for a subset of vocabulary ids (needs lse for every token)."""
    H = _f64(H)
    Wv = _f64(W)[np.asarray(vocab_rows)]
    y = np.asarray(y, dtype=np.int64)
    lse = _f64(lse)
    g = _f64(g)
    vr = np.asarray(vocab_rows, dtype=np.int64)
    out = np.zeros((len(vr), H.shape[1]), dtype=np.float64)
    for a in range(0, H.shape[0], row_chunk):
        b = min(H.shape[0], a + row_chunk)
        z = H[a:b] @ Wv.T
        dz = -np.exp(z - lse[a:b, None])
        dz += (y[a:b, None] == vr[None, :])
        dz *= g[a:b, None]
        out += dz.T @ H[a:b]
    return out


def token_entropy(H, W, row_chunk=64):
    """Return H float64[T]: -sum_v p log p of each row's softmax (0 log 0 = 0)."""
    H = _f64(H)
    W = _f64(W)
    T = H.shape[0]
    out = np.empty(T, dtype=np.float64)
    for a in range(0, T, row_chunk):
        b = min(T, a + row_chunk)
        z = H[a:b] @ W.T
        m = z.max(axis=1)
        e = np.exp(z - m[:, None])
        p = e / e.sum(axis=1)[:, None]
        logp = np.where(p > 0, np.log(np.where(p > 0, p, 1.0)), 0.0)
        out[a:b] = -(p * logp).sum(axis=1)
    return out
