"""Oracle: tensor-parallel LM head with vocabulary-parallel cross-entropy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's model ends in RMSNorm -> linear (h x v, untied from the embedding)
-> softmax / cross-entropy kept in FP32 (Sec. 3, "LM Head" in Sec. 3.2).  With
tensor parallelism the vocabulary is split over t ranks; a rank holds rows
[vocab_start, vocab_start + v_t) of the head weight.  The statistics that the
vocabulary-parallel loss all-reduces across ranks arrive as inputs:
``peer_lse`` (log-sum-exp of the other ranks' logits, per token) and
``peer_target_logit`` (the target's logit when another rank owns it).

Readings: logits are stored in bf16 and every later quantity is computed from
the stored logits in float (the softmax statistics in FP32 in the library,
float64 here); loss_i = LSE_i - z_i; dlogits = (softmax - onehot) * grad_scale
stored in bf16; the hidden-state gradient is stored in bf16, the weight
gradient is a float accumulator.
"""
import numpy as np

from .bf16 import round_bf16


def lm_head_xent(hidden, w_lm, targets, vocab_start=0, peer_lse=None,
                 peer_target_logit=None, grad_scale=1.0, exact=False):
    """hidden [N, h], w_lm [v_t, h], targets [N] global ids.
    Returns dict(loss [N], lse [N], logits, dlogits, d_hidden [N, h], d_w [v_t, h])."""
    rnd = (lambda a: a) if exact else round_bf16
    n, v_t = hidden.shape[0], w_lm.shape[0]
    logits = rnd(hidden @ w_lm.T)
    m = logits.max(axis=1)
    lse = m + np.log(np.exp(logits - m[:, None]).sum(axis=1))
    if peer_lse is not None:
        lse = np.logaddexp(lse, peer_lse)
    local = np.asarray(targets) - vocab_start
    own = (local >= 0) & (local < v_t)
    rows = np.arange(n)
    z = np.where(own, logits[rows, np.clip(local, 0, v_t - 1)], 0.0)
    if not own.all():
        if peer_target_logit is None:
            raise ValueError("a target outside this shard needs peer_target_logit")
        z = np.where(own, z, peer_target_logit)
    loss = lse - z
    g = np.exp(logits - lse[:, None])
    g[rows[own], local[own]] -= 1.0
    dlogits = rnd(g * grad_scale)
    return dict(loss=loss, lse=lse, logits=logits, dlogits=dlogits,
                d_hidden=rnd(dlogits @ w_lm), d_w=dlogits.T @ hidden)
