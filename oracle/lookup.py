"""Exhaustive top-1 cosine search over the prompt-embedding cache.

Test infrastructure only (see the package docstring).

Approximate caching retrieves the most similar cached prompt by similarity
search over prompt embeddings held in a vector database (Sec. 2.1; Sec. 4.5;
Sec. 4.7). Here the similarity is cosine, computed exhaustively:
score_i = (q . c_i) / (|q| |c_i|) with the fp16 inputs widened to fp64, and the
result is argmax_i score_i with ties going to the lowest index.
"""

import numpy as np


def cosine_scores(query, cache):
    """fp64 cosine similarity of query [dim] against every row of cache [n, dim].
    A zero-norm row has no defined cosine and scores -inf (it never wins)."""
    q = np.asarray(query, dtype=np.float64)
    c = np.asarray(cache, dtype=np.float64)
    norms = np.linalg.norm(c, axis=1)
    out = np.full(c.shape[0], -np.inf)
    ok = norms > 0
    out[ok] = (c[ok] @ q) / (norms[ok] * np.linalg.norm(q))
    return out


def top1(query, cache):
    """(index, score) of the best row; np.argmax returns the first maximum, i.e. the
    lowest index among equal scores."""
    s = cosine_scores(query, cache)
    i = int(np.argmax(s))
    return i, float(s[i])


def top2_gap(query, cache):
    """Score gap between the best and the second-best row (inf if n < 2)."""
    s = cosine_scores(query, cache)
    if s.size < 2:
        return float("inf")
    a = np.partition(s, -2)[-2:]
    return float(a[1] - a[0])
