"""The SpS loop (Algorithm 2) and auto-regressive sampling (Algorithm 1).

Oracle (test infrastructure only). Every model call is a full causal
recompute of the whole sequence (model.forward_full): slow and obviously
correct, with no cache bookkeeping to get wrong.

Reading of Algorithm 2 (the printed loop increments n inside the accept loop
while also indexing by n + t, and the bonus-token line is garbled):
  * n is fixed while the K drafts are tested; afterwards the sequence grows
    by a + 1 tokens, where a is the number of accepted drafts;
  * a rejection emits the resampled token and ends the loop (at least one
    token per loop);
  * when all K drafts are accepted, the bonus token is drawn from the target
    distribution that follows x~_K, the (K+1)-th row of the scoring call;
  * T is a minimum length, so the last loop may overshoot; the output is
    truncated to exactly n_new tokens (a prefix of a target-distributed
    sequence is target distributed).
Randomness per sequence b and loop index l comes from Philox (see philox.py):
draft position t uses purpose DRAFT at j = t - 1, its accept test uses
purpose ACCEPT at j = t - 1, and the final draw uses purpose RESAMPLE at
j = 0. ArS is the K = 0 case: every token is the "bonus" draw from q with
purpose RESAMPLE, so ArS and SpS consume the random stream differently, as
the paper notes.
"""
import numpy as np

from . import philox
from .accept import accept_resample_one
from .model import forward_full
from .sampling import softmax, to_weights, categorical


def probs_fp32(logits, temperature):
    """Distribution handed to the sampler: fp64 softmax, stored as fp32."""
    return softmax(logits, temperature).astype(np.float32)


def sps_generate_one(tspec, tW, dspec, dW, prompt, n_new, K, temperature, seed, b=0, loop0=0, truncate=True,
                     trace=None):
    """Generate n_new tokens for one sequence (batch index b in the RNG).

    Returns (tokens, accepted) where accepted lists a per loop. The SpS
    state at a loop boundary is the token sequence and the loop index, so a
    run can stop there (truncate=False keeps every token of the last loop)
    and resume: the next call takes prompt + the tokens so far and loop0 =
    the loops done. If trace is a list, each loop appends a dict of its
    drafts, p rows, q rows, uniforms and outcome.
    """
    seq = [int(t) for t in prompt]
    out = []
    accepted = []
    loop = loop0
    while len(out) < n_new:
        drafts, ps = [], []
        if K > 0:
            ud = philox.uniforms(seed, loop, philox.PURPOSE_DRAFT, b + 1, K)[b]
        for t in range(K):
            logits = forward_full(dspec, dW, np.array([seq + drafts]))[0, -1]
            p = probs_fp32(logits, temperature)
            x, _ = categorical(to_weights(p), ud[t])
            drafts.append(x)
            ps.append(p)
        n = len(seq)
        logits = forward_full(tspec, tW, np.array([seq + drafts]))[0, n - 1:n + K]
        q = probs_fp32(logits, temperature)
        r = philox.uniforms(seed, loop, philox.PURPOSE_ACCEPT, b + 1, K)[b] if K else np.zeros(0, np.float32)
        u = philox.uniforms(seed, loop, philox.PURPOSE_RESAMPLE, b + 1, 1)[b]
        unif = np.concatenate([r, u])
        p_arr = np.array(ps, dtype=np.float32).reshape(K, q.shape[-1])
        toks, a, _ = accept_resample_one(p_arr, q, drafts, unif)
        if trace is not None:
            trace.append({"loop": loop, "drafts": list(drafts), "ud": ud[:K] if K else None, "p": p_arr, "q": q,
                          "unif": unif, "a": a, "tokens": toks})
        seq += toks
        out += toks
        accepted.append(a)
        loop += 1
    return (out[:n_new] if truncate else out), accepted


def ars_generate_one(tspec, tW, prompt, n_new, temperature, seed, b=0):
    """Algorithm 1: one target call and one draw per token (the K = 0 loop)."""
    return sps_generate_one(tspec, tW, None, None, prompt, n_new, 0, temperature, seed, b)
