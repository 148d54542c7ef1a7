"""Oracle: streaming chunk attention against a KV cache (test infrastructure).

Definitions followed (arXiv 2607.00712):

* Sec. 2, Eq. 3 (KV injection): the queries are the current chunk only; the
  keys/values are the cached past followed by the current chunk. So with a
  cache holding ``cache_len`` keys, the last ``n_q`` rows of the cache are the
  current chunk and every query sees every key of the set it attends to (no
  mask inside a chunk).
* Sec. 2, the remark after Eq. 3: baseline models keep only the most recent
  frames, i.e. a sliding window at the cache tail.
* Sec. 3.4, Eq. 7-8: the local context is the sink prefix together with the
  current (most recent) keys; the history is everything in between; the full
  set is their disjoint union.
* Sec. 3.4, Eq. 9-10: each branch is ordinary softmax attention returning the
  output and its log-sum-exp.
* Sec. 3.4, Eq. 11-12: the full output is the LSE-weighted combination of the
  two branches.

Readings where the paper is silent:

* the local set is ``[0, min(s, N)) U [max(N - w, 0), N)`` for a window of
  ``w`` keys and a sink of ``s`` keys; the history is ``[s, N - w)`` when that
  is non-empty;
* logits are scaled by ``1/sqrt(head_dim)`` unless a scale is given;
* LSE uses the natural logarithm; an empty key set has LSE = -inf and a zero
  output, which makes the fusion of Eq. 11-12 return the other branch.

Everything is computed in float64 straight from the definition: scores,
row max, exponentials, normaliser, probabilities, weighted sum. Queries are
processed in blocks only to bound memory; nothing is reordered.
"""

import math

import numpy as np

_QUERY_BLOCK = 256


def visible_key_sets(cache_len, window, sink_len=0):
    """Index sets of Sec. 3.4, Eq. 7-8 for a cache of ``cache_len`` keys.

    Returns ``(local, hist)``, two sorted int64 arrays whose disjoint union is
    ``range(cache_len)`` (the full set of Eq. 8's last line).
    """
    n = int(cache_len)
    w = int(window)
    s = int(sink_len)
    if n < 0 or w < 0 or s < 0:
        raise ValueError("cache_len, window and sink_len must be >= 0")
    in_local = np.zeros(n, dtype=bool)
    in_local[: min(s, n)] = True          # sink frame(s): the cache prefix
    in_local[max(n - w, 0):] = True       # current / most recent keys
    local = np.flatnonzero(in_local).astype(np.int64)
    hist = np.flatnonzero(~in_local).astype(np.int64)
    return local, hist


def attend(q, k, v, keys, scale, return_probs=False):
    """Softmax attention of one head over an explicit key set (Eq. 9-10).

    q: [n_q, d] ; k, v: [N, d] ; keys: int index array into the rows of k/v.
    Returns ``(o [n_q, d], lse [n_q])`` in float64, and the probability
    matrix ``p [n_q, |keys|]`` when ``return_probs`` is set.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    keys = np.asarray(keys, dtype=np.int64)
    n_q, d = q.shape
    o = np.zeros((n_q, v.shape[1]), dtype=np.float64)
    lse = np.full(n_q, -np.inf, dtype=np.float64)
    probs = np.zeros((n_q, keys.size), dtype=np.float64) if return_probs else None
    if keys.size == 0:
        return (o, lse, probs) if return_probs else (o, lse)
    ks = k[keys]
    vs = v[keys]
    for r0 in range(0, n_q, _QUERY_BLOCK):
        r1 = min(r0 + _QUERY_BLOCK, n_q)
        s = (q[r0:r1] @ ks.T) * scale                 # logits
        m = s.max(axis=1, keepdims=True)              # row max
        e = np.exp(s - m)                             # shifted exponentials
        l = e.sum(axis=1, keepdims=True)              # normaliser
        p = e / l                                     # softmax rows
        o[r0:r1] = p @ vs
        lse[r0:r1] = m[:, 0] + np.log(l[:, 0])
        if return_probs:
            probs[r0:r1] = p
    return (o, lse, probs) if return_probs else (o, lse)


def lse_merge(o_a, lse_a, o_b, lse_b):
    """Log-sum-exp fusion of two disjoint branches (Sec. 3.4, Eq. 11-12).

    ``o_*`` are [..., d] outputs, ``lse_*`` the matching [...] log-sum-exps.
    Eq. 11 is evaluated as ``m + log(exp(a - m) + exp(b - m))`` with
    ``m = max(a, b)`` so that it does not overflow; two empty branches give
    LSE = -inf and a zero output.
    """
    lse_a = np.asarray(lse_a, dtype=np.float64)
    lse_b = np.asarray(lse_b, dtype=np.float64)
    o_a = np.asarray(o_a, dtype=np.float64)
    o_b = np.asarray(o_b, dtype=np.float64)
    m = np.maximum(lse_a, lse_b)
    both_empty = np.isneginf(m)
    m_safe = np.where(both_empty, 0.0, m)
    with np.errstate(divide="ignore"):
        lse = m_safe + np.log(np.exp(lse_a - m_safe) + np.exp(lse_b - m_safe))
    lse = np.where(both_empty, -np.inf, lse)
    lse_safe = np.where(both_empty, 0.0, lse)
    wa = np.where(both_empty, 0.0, np.exp(lse_a - lse_safe))
    wb = np.where(both_empty, 0.0, np.exp(lse_b - lse_safe))
    o = wa[..., None] * o_a + wb[..., None] * o_b
    return o, lse


def chunk_attention(q, k_cache, v_cache, cache_len, window, n_heads,
                    sink_len=0, scale=None, branches=("full", "local", "hist"),
                    query_rows=None):
    """Attention of one chunk's queries against one layer's KV cache.

    Layouts (row-major, heads concatenated as in the projection input):
      q        [n_q, n_heads * d]
      k_cache  [>= cache_len, n_heads * d]   (rows beyond cache_len ignored)
      v_cache  [>= cache_len, n_heads * d]

    ``query_rows`` optionally restricts the computation to a subset of query
    rows (used to spot-check very large chunks one row at a time); the
    outputs then have ``len(query_rows)`` rows.

    Returns ``{branch: (o [rows, n_heads * d], lse [n_heads, rows])}`` for each
    requested branch among "full" (all keys), "local" (Eq. 7) and "hist"
    (Eq. 8), all in float64.
    """
    q = np.asarray(q)
    n_q, hd = q.shape
    if hd % n_heads:
        raise ValueError("hidden size is not a multiple of n_heads")
    d = hd // n_heads
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(d)
    n = int(cache_len)
    k_cache = np.asarray(k_cache)[:n]
    v_cache = np.asarray(v_cache)[:n]
    rows = np.arange(n_q) if query_rows is None else np.asarray(query_rows, dtype=np.int64)
    local, hist = visible_key_sets(n, window, sink_len)
    key_sets = {"full": np.arange(n, dtype=np.int64), "local": local, "hist": hist}
    out = {}
    for name in branches:
        o = np.zeros((rows.size, hd), dtype=np.float64)
        lse = np.zeros((n_heads, rows.size), dtype=np.float64)
        for h in range(n_heads):
            cols = slice(h * d, (h + 1) * d)
            o_h, lse_h = attend(q[rows, cols], k_cache[:, cols], v_cache[:, cols],
                                key_sets[name], scale)
            o[:, cols] = o_h
            lse[h] = lse_h
        out[name] = (o, lse)
    return out
