"""Oracle: the two ends of the model on one (TP, CP) shard, forward and backward:
the vocabulary-parallel embedding and the LM-head block (final RMSNorm ->
linear -> FP32 softmax cross-entropy), as the activation terms of Sec. 3.2
describe them.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Embedding (Sec. 3.2, the embedding term): the input is the int64 token ids.
With TP the table is split by vocabulary: a rank holds rows [v0, v0 + v_t) and
produces, for every token of its CP chunk, the table row when the id falls in
its range and zeros otherwise; the sum over the TP group (a reduce-scatter
under sequence parallelism) gives each rank its own rows.  As in the layer
oracle, the peers' partial sums for the own rows arrive as ``receipt`` and this
rank's partial rows for the peers leave as ``send``.  The backward adds, for
every token whose id is in range, the gathered output gradient to that row of
the table's gradient.

LM-head block (Sec. 3.2, the LM-head term 4sbh(1 + v/h)): xn = RMSNorm(x) on
the own rows (the "2sbh for the output RMSNorm" is x, the "2sbh for the output
linear layer" is xn), all-gathered over the TP group, logits = xn W^T over the
rank's vocabulary shard, kept in FP32 ("4sbv"), cross-entropy as in
``lm_head.lm_head_xent`` with the statistics of the other shards as inputs.
The FP32 tensor the backward needs is the softmax; the backward forms
dlogits = (softmax - onehot) * grad_scale.

Readings (the rounding points are where the library stores a tensor):
  * xn, dlogits, d(xn) and dx are stored in bf16; logits, softmax and loss in
    FP32 (float64 here); weight and gain gradients are float accumulators.
  * d(xn) of the own rows is bf16(own partial + the peers' partials received);
    the partial rows for the peers are sent as bf16.
  * the embedding output of an own row is bf16(partial + receipt); exactly
    one rank holds a token's row, so the sum is exact.
``exact=True`` drops every rounding (for finite differences).
"""
import numpy as np

from .bf16 import round_bf16
from .layer import gather, rmsnorm, rmsnorm_bwd, split_own
from .lm_head import lm_head_xent


def embedding_forward(sh, w, ids, vocab_start, receipt=None, exact=False):
    """w [v_t, h] table shard, ids [b, s_c] global ids of the rank's CP tokens.
    Returns dict(partial [b, s_c, h], own [b, s_sp, h], send [b, (t-1) s_sp, h])."""
    rnd = (lambda a: a) if exact else round_bf16
    v_t = w.shape[0]
    local = np.asarray(ids) - vocab_start
    hit = (local >= 0) & (local < v_t)
    partial = np.where(hit[..., None], w[np.clip(local, 0, v_t - 1)], 0.0)
    own, send = split_own(sh, partial)
    if receipt is not None:
        own = own + receipt
    return dict(partial=partial, own=rnd(own), send=rnd(send))


def embedding_backward(sh, ids, dy_own, dy_peer, v_t, vocab_start):
    """Table-shard gradient [v_t, h]: the gathered output gradient of every
    token summed into the row of its id, for the ids in this rank's range."""
    dy = gather(sh, dy_own, dy_peer)
    local = (np.asarray(ids) - vocab_start).reshape(-1)
    dy = dy.reshape(-1, dy.shape[-1])
    dw = np.zeros((v_t, dy.shape[-1]))
    for m, j in enumerate(local):
        if 0 <= j < v_t:
            dw[j] += dy[m]
    return dw


def lm_head_forward(sh, x, gain, w_lm, targets, vocab_start, peer_xn=None, peer_lse=None,
                    peer_target_logit=None, exact=False):
    """x [b, s_sp, h] own rows (the last layer's output), gain [h], w_lm [v_t, h],
    targets [b, s_c].  Returns dict(xn [b, s_sp, h], logits, probs [b*s_c, v_t],
    lse, loss [b*s_c])."""
    rnd = (lambda a: a) if exact else round_bf16
    xn = rnd(rmsnorm(x, gain, sh.eps))
    full = gather(sh, xn, peer_xn).reshape(-1, x.shape[-1])
    r = lm_head_xent(full, w_lm, np.asarray(targets).reshape(-1), vocab_start,
                     None if peer_lse is None else np.asarray(peer_lse).reshape(-1),
                     None if peer_target_logit is None else np.asarray(peer_target_logit).reshape(-1),
                     exact=True)
    probs = np.exp(r["logits"] - r["lse"][:, None])
    return dict(xn=xn, gathered=full, logits=r["logits"], probs=probs, lse=r["lse"], loss=r["loss"])


def lm_head_backward(sh, x, gain, w_lm, targets, vocab_start, fw, grad_scale=1.0, peer_dxn=None,
                     exact=False):
    """Backward of lm_head_forward for d(sum of loss * grad_scale).  Returns
    dict(dlogits, dx [b, s_sp, h], d_gain [h], d_w [v_t, h], send [b, (t-1) s_sp, h])."""
    rnd = (lambda a: a) if exact else round_bf16
    v_t = w_lm.shape[0]
    g = fw["probs"].copy()
    local = np.asarray(targets).reshape(-1) - vocab_start
    own = (local >= 0) & (local < v_t)
    g[np.nonzero(own)[0], local[own]] -= 1.0
    dlogits = rnd(g * grad_scale)
    d_full = (dlogits @ w_lm).reshape(x.shape[0], -1, x.shape[-1])
    d_own, d_peer = split_own(sh, d_full)
    if peer_dxn is not None:
        d_own = d_own + peer_dxn
    d_xn = rnd(d_own)
    dx, d_gain = rmsnorm_bwd(x, gain, sh.eps, d_xn)
    return dict(dlogits=dlogits, d_xn=d_xn, dx=rnd(dx), d_gain=d_gain, d_w=dlogits.T @ fw["gathered"],
                send=rnd(d_peer))
