"""Modified rejection sampling: the accept / resample / bonus step of SpS.

Oracle (test infrastructure only). Notation follows the paper: q is the
TARGET model, p is the DRAFT model.

Given, for one sequence, the K draft tokens x~_1..x~_K, the draft
distributions p_1..p_K they were sampled from, the K+1 target distributions
q_1..q_{K+1} from one parallel scoring call, K accept uniforms r_1..r_K and
one uniform u for the final draw (Algorithm 2; Modified Rejection Sampling
section):

1. Left to right, accept x~_t with probability min(1, q_t(x~_t) / p_t(x~_t)).
   The test r < min(1, rho/pi) with rho = q_t(x~_t), pi = p_t(x~_t) is taken
   as  r * pi < rho  evaluated in fp64. For fp32 r and pi the product is
   exact in fp64, so the decision is exact for the given fp32 values and
   needs no division. pi = 0 accepts iff rho > 0. The first rejection at
   position t fixes a = t - 1 accepted tokens and stops the scan.
2. If a < K, draw the replacement for x~_{a+1} from (q_{a+1} - p_{a+1})_+,
   the normalised positive part (Modified Rejection Sampling section). In
   fixed point the weights are max(0, floor(q 2^32) - floor(p 2^32)). Their
   total is zero only through rounding (exact arithmetic makes the event
   have probability zero); the draw then falls back to q_{a+1}.
3. If a == K, every draft was accepted and the bonus token is drawn from
   q_{K+1}, the distribution that follows the last draft (Algorithm 2, final
   step), giving K+1 tokens.
4. Emit x~_1..x~_a followed by the drawn token: between 1 and K+1 tokens.

Theorem 1 shows step 1 + step 2 reproduce q exactly; the tests check the
sequential law by exact enumeration and by chi-square.

Error handling (defined outputs, no exceptions): a draft token outside
[0, V) is treated as rejected at its position and sets FLAG_BAD_TOKEN; a
draw whose weights are all zero returns token 0 and sets FLAG_EMPTY. The
paper assumes valid distributions; a sequence whose inputs are not -- a
target row marked as having non-finite logits, a NaN or infinite value
among the gathered q_t(x~_t), p_t(x~_t) (every t with a valid draft
token), or among the entries of the rows the final draw reads -- is given
a = 0 and token 0 and sets FLAG_NONFINITE.
"""
import numpy as np

from . import philox
from .sampling import to_weights, categorical

FLAG_BAD_TOKEN = 1
FLAG_EMPTY = 2
FLAG_NONFINITE = 8


def _finite(x):
    return bool(np.all(np.isfinite(np.asarray(x, dtype=np.float32))))


def accept_test(r, pi, rho):
    """The exact accept decision r < min(1, rho / pi) on fp32 inputs."""
    return float(np.float32(r)) * float(np.float32(pi)) < float(np.float32(rho))


def residual_weights(q_row, p_row):
    """Fixed-point weights of (q - p)_+ : max(0, floor(q 2^32) - floor(p 2^32))."""
    wq = to_weights(q_row).astype(np.int64)
    wp = to_weights(p_row).astype(np.int64)
    return np.maximum(wq - wp, 0).astype(np.uint64)


def accept_resample_one(p, q, drafts, unif, bad_rows=None):
    """One sequence. p: [K][V], q: [K+1][V] fp32; drafts: [K]; unif: [K+1];
    bad_rows: optional [K+1] bools, target rows whose logits were
    non-finite.

    Returns (tokens, a, flags) where tokens has length a + 1.
    """
    K = len(drafts)
    V = q.shape[-1]
    flags = 0
    nonfinite = bad_rows is not None and bool(np.any(bad_rows))
    for t in range(K):                     # every gathered value is checked
        x = int(drafts[t])
        if 0 <= x < V and not (_finite(q[t][x]) and _finite(p[t][x])):
            nonfinite = True
    a = K
    for t in range(K):                     # draft position t+1 in the paper
        x = int(drafts[t])
        if x < 0 or x >= V:
            flags |= FLAG_BAD_TOKEN
            a = t
            break
        if not accept_test(unif[t], p[t][x], q[t][x]):
            a = t
            break
    if not nonfinite:
        if a < K:
            nonfinite = not (_finite(q[a]) and _finite(p[a]))
            w = residual_weights(q[a], p[a])
            if int(w.sum(dtype=np.uint64)) == 0:
                w = to_weights(q[a])
        else:
            nonfinite = not _finite(q[K])
            w = to_weights(q[K])
    if nonfinite:
        return [0], 0, flags | FLAG_NONFINITE
    y, ok = categorical(w, unif[K])
    if not ok:
        flags |= FLAG_EMPTY
    return [int(v) for v in drafts[:a]] + [y], a, flags


def accept_resample(p_draft, q_target, draft_tokens, unif, bad_rows=None):
    """Batched: p_draft [B][K][V], q_target [B][K+1][V], draft_tokens [B][K],
    unif [B][K+1] (r_1..r_K, then u), bad_rows [B][K+1] or None.

    Returns out_tokens [B][K+1] int32 (entries after the a+1 emitted tokens
    are -1), n_accepted [B] int32, flags [B] int32.
    """
    p_draft = np.asarray(p_draft, dtype=np.float32)
    q_target = np.asarray(q_target, dtype=np.float32)
    draft_tokens = np.asarray(draft_tokens)
    unif = np.asarray(unif, dtype=np.float32)
    B, K1, _ = q_target.shape
    K = K1 - 1
    out = np.full((B, K + 1), -1, dtype=np.int32)
    n_acc = np.zeros(B, dtype=np.int32)
    flags = np.zeros(B, dtype=np.int32)
    for b in range(B):
        toks, a, f = accept_resample_one(p_draft[b] if K else np.zeros((0, q_target.shape[-1]), np.float32),
                                         q_target[b], draft_tokens[b][:K], unif[b],
                                         None if bad_rows is None else bad_rows[b])
        out[b, :a + 1] = toks
        n_acc[b] = a
        flags[b] = f
    return out, n_acc, flags


def philox_uniforms(seed, loop, B, K):
    """The [B][K+1] uniforms one SpS loop uses: r_t from purpose ACCEPT at
    j = t - 1, then u from purpose RESAMPLE at j = 0."""
    r = philox.uniforms(seed, loop, philox.PURPOSE_ACCEPT, B, K)
    u = philox.uniforms(seed, loop, philox.PURPOSE_RESAMPLE, B, 1)
    return np.concatenate([r, u], axis=1)
