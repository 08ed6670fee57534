"""Decode attention definitions in fp64 (test infrastructure only).

Notation of Sec. 3.1-3.3: one query q (d,), n keys k_i and values v_i (rows
of K, V), scaled logits q k_i / sqrt(d).  All functions take float64 arrays.
"""
import numpy as np


def logits(q: np.ndarray, K: np.ndarray) -> np.ndarray:
    """q k_i^T / sqrt(d) for every row of K (Sec. 2.1, Eq. 2)."""
    d = q.shape[-1]
    return (K @ q) / np.sqrt(d)


def softmax_weights(l: np.ndarray) -> np.ndarray:
    """Attention scores s_i = exp(l_i) / sum_j exp(l_j), computed with a max
    shift so that nothing overflows (the shift cancels in the ratio)."""
    e = np.exp(l - np.max(l))
    return e / e.sum()


def dense_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """o = sum_i s_i v_i with s = softmax(q K^T / sqrt(d))  (Eq. 2).

    Eq. 1 prints softmax(exp(Q K^T / sqrt(d))) V, an extra exp; the decode
    form of Eq. 2 is the one used here."""
    return softmax_weights(logits(q, K)) @ V


def sparse_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, idx) -> np.ndarray:
    """o~(I) = sum_{i in I} s~_i v_i, softmax renormalised over I  (Eq. 3)."""
    idx = np.asarray(idx, dtype=np.int64)
    return dense_attention(q, K[idx], V[idx])


def cumulative_score(q: np.ndarray, K: np.ndarray, idx) -> float:
    """p(I) = sum_{i in I} s_i with s the full softmax  (Eq. 5)."""
    s = softmax_weights(logits(q, K))
    return float(s[np.asarray(idx, dtype=np.int64)].sum())


def attention_distance(q: np.ndarray, K: np.ndarray, V: np.ndarray, idx) -> float:
    """epsilon(I) = || o - o~(I) ||  (Eq. 4)."""
    return float(np.linalg.norm(dense_attention(q, K, V) - sparse_attention(q, K, V, idx)))


def error_bound(q: np.ndarray, K: np.ndarray, V: np.ndarray, idx) -> float:
    """Right-hand side of Eq. 6: 2 (1 - p(I)) max_i ||v_i||  (Appendix A)."""
    p = cumulative_score(q, K, idx)
    return 2.0 * (1.0 - p) * float(np.max(np.linalg.norm(V, axis=1)))


def optimal_selection(q: np.ndarray, K: np.ndarray, P: float) -> np.ndarray:
    """The smallest index set reaching cumulative score P (Sec. 1 and 3.4):
    tokens in descending order of attention score until the running sum of
    scores reaches P.  Ties in score are taken in ascending index order.
    Returns the selected indices in selection order."""
    s = softmax_weights(logits(q, K))
    order = np.lexsort((np.arange(len(s)), -s))
    c = 0.0
    for k, i in enumerate(order, start=1):
        c += s[i]
        if c >= P:
            return order[:k]
    return order
