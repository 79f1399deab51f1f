"""Top-k and nucleus (top-p) modifiers of the draft and target distributions.

Oracle (test infrastructure only).

The paper applies the usual sampling modifiers -- temperature, top-k and
nucleus -- to the probabilities before the rejection step, and its headline
runs use nucleus sampling (Modified Rejection Sampling section, closing
paragraph; Table 1 and its caption: nucleus 0.8 on XSum, 0.95 with
temperature 0.8 on HumanEval). Theorem 1 then holds for the modified
distributions: the draft must be sampled from exactly the modified p that
acceptance uses, and the output follows the modified q. The paper gives no
formula for the modifiers; they are read here as follows (both the GPU
path and this oracle):

* order: temperature first (the softmax), then top-k, then nucleus on what
  top-k kept -- the same for p and q;
* ranking: entries are ranked by their fixed-point draw weight
  w_i = floor(x_i 2^32) (the weight the categorical draw uses), larger
  first, equal weights by lower index first. This is a total order, so the
  kept set of every modifier is unique and needs no floating-point sum;
* top-k (1 <= k < V): the first k entries of the ranking;
* nucleus (0 <= p < 1): among the entries top-k kept (all entries if top-k
  is off), with W_k their weight total, the shortest prefix of the ranking
  whose weight sum reaches floor(floor(p 2^24) W_k / 2^24) -- the same
  grid arithmetic as the draw threshold -- and at least one entry;
* renormalisation: S = the exact integer weight total of the kept entries,
  s = fp32(S) * 2^-32 with fp32(S) rounded to nearest (ties to even) once,
  x'_i = fp32(x_i / s) for kept entries and 0 elsewhere;
* a row is left unchanged when both modifiers are off (k <= 0 or k >= V,
  and p >= 1) or when the kept weights sum to zero.

Every step is integer arithmetic or one correctly rounded fp32 operation, so
a parallel implementation agrees with this one bit for bit. Ranking on w
instead of x differs from ranking on exact probabilities only between
entries closer than 2^-32.
"""
import numpy as np

from .sampling import grid_index, to_weights


def rank_order(w):
    """Indices sorted by weight (descending), equal weights by lower index."""
    w = np.asarray(w, dtype=np.uint64).astype(np.int64)
    return np.lexsort((np.arange(w.shape[0]), -w))


def active(V, top_k, top_p):
    return (1 <= int(top_k) < V) or float(top_p) < 1.0


def kept_count(w_ranked, top_k, top_p):
    """Number of leading entries of the ranking the modifiers keep.

    w_ranked: Python ints, the weights in ranking order.
    """
    V = len(w_ranked)
    n = int(top_k) if 1 <= int(top_k) < V else V
    if float(top_p) < 1.0:
        Wk = sum(w_ranked[:n])
        target = (grid_index(np.float32(max(float(top_p), 0.0))) * Wk) >> 24
        acc, j = 0, 0
        while True:                           # shortest prefix reaching target, >= 1 entry
            acc += w_ranked[j]
            j += 1
            if acc >= target:
                break
        n = j
    return n


def fp32_of_int(S):
    """The fp32 value nearest to the non-negative integer S (ties to even)."""
    S = int(S)
    e = S.bit_length()
    if e <= 24:
        return np.float32(S)
    shift = e - 24
    q, r = S >> shift, S & ((1 << shift) - 1)
    half = 1 << (shift - 1)
    if r > half or (r == half and (q & 1)):
        q += 1
    return np.float32(np.ldexp(np.float64(q), shift))


def kept_mask(x, top_k, top_p):
    """Boolean mask of the entries the modifiers keep (all True if inactive)."""
    x = np.asarray(x, dtype=np.float32)
    V = x.shape[-1]
    if not active(V, top_k, top_p):
        return np.ones(V, dtype=bool)
    w = to_weights(x)
    order = rank_order(w)
    n = kept_count([int(w[i]) for i in order], top_k, top_p)
    mask = np.zeros(V, dtype=bool)
    mask[order[:n]] = True
    return mask


def modify(x, top_k=0, top_p=1.0):
    """The modified distribution of one fp32 probability row x (see module doc)."""
    x = np.asarray(x, dtype=np.float32)
    V = x.shape[-1]
    if not active(V, top_k, top_p):
        return x.copy()
    mask = kept_mask(x, top_k, top_p)
    w = to_weights(x)
    S = sum(int(v) for v in w[mask])
    if S == 0:
        return x.copy()
    s = np.float32(fp32_of_int(S) * np.float32(2.0 ** -32))
    out = np.zeros(V, dtype=np.float32)
    out[mask] = x[mask] / s                   # fp32 division, correctly rounded
    return out


def modify_rows(x, top_k=0, top_p=1.0):
    """modify() applied to every row of an [..., V] array."""
    x = np.asarray(x, dtype=np.float32)
    flat = x.reshape(-1, x.shape[-1])
    out = np.stack([modify(r, top_k, top_p) for r in flat])
    return out.reshape(x.shape)
