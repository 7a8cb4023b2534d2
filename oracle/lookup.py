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


def cosine_scores_batch(queries, cache):
    """fp64 cosine similarity of every query row [nq, dim] against every cache row
    [n, dim]: [nq, n]. Zero-norm rows score -inf; a zero query's row is all nan."""
    q = np.atleast_2d(np.asarray(queries, dtype=np.float64))
    c = np.asarray(cache, dtype=np.float64)
    cn = np.linalg.norm(c, axis=1)
    qn = np.linalg.norm(q, axis=1)
    out = np.full((q.shape[0], c.shape[0]), -np.inf)
    ok = cn > 0
    out[:, ok] = (q @ c[ok].T) / cn[ok][None, :]
    with np.errstate(divide="ignore", invalid="ignore"):
        out = out / qn[:, None]
    out[qn == 0] = np.nan
    return out


def top1_batch(queries, cache):
    """Batched search (approximate caching serves many prompts against one cache,
    Sec. 2.1; Sec. 4.5): for every query row, the row of maximal cosine exactly as
    `top1`, ties to the lowest index. A zero query has no defined cosine and gets
    (-1, nan); so does a query against a cache of zero rows only.
    Returns (indices [nq] int64, scores [nq] fp64)."""
    s = cosine_scores_batch(queries, cache)
    idx = np.full(s.shape[0], -1, np.int64)
    score = np.full(s.shape[0], np.nan)
    for j in range(s.shape[0]):
        if not np.isfinite(s[j]).any():
            continue
        idx[j] = int(np.argmax(s[j]))
        score[j] = float(s[j, idx[j]])
    return idx, score


def select_k(scores, thresholds, levels):
    """Approximation level chosen from the similarity of the retrieved prompt (Sec. 2.1:
    the cached state to resume from is picked by how similar the cached prompt is; the
    more similar, the more iterations may be skipped). Reading: a monotone threshold
    table with thresholds t_1 < ... < t_L and levels K_0 <= ... <= K_L;
    a retrieved cosine s gets K_j with j = #{i : s >= t_i}, compared in the precision the
    score is given in (fp32 on both sides). A query that retrieved nothing (index -1,
    score nan) gets K = 0: there is no cached state to resume from.
    scores [nq] fp32, thresholds [L], levels [L + 1] -> K [nq] int32."""
    s = np.asarray(scores, dtype=np.float32)
    t = np.asarray(thresholds, dtype=np.float32)
    lv = [int(v) for v in levels]
    if len(lv) != t.size + 1:
        raise ValueError("levels must have one entry more than thresholds")
    out = np.zeros(s.size, np.int32)
    for q in range(s.size):
        if np.isnan(s[q]):
            continue
        j = 0
        for i in range(t.size):
            if s[q] >= t[i]:
                j = i + 1
        out[q] = lv[j]
    return out
