"""Closed-form per-GPU memory of 4D-parallel Llama training (Sec. 3, Eqs. 1-18).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Every quantity is an exact rational (``fractions.Fraction``) so that a table
cell can be compared to the byte.  Symbols follow the paper's variable table:
a heads, k key-value heads, b micro-batch, h hidden, d data-parallel size,
h_ffn FFN hidden, L layers, p pipeline size, s sequence, t tensor size,
c context size, v vocabulary.

Readings where the text leaves a choice:
  * p == 1: the single stage holds the embedding, the LM head, the final
    RMSNorm and all L layers, so the parameter count is 2hv/t + h + L*ell
    (Eq. 6 with the last-stage terms of Eq. 9); the printed total Eq. 18 shows
    only the first-stage form hv/t, which does not reproduce the paper's own
    tables for PP = 1.  For p > 1 the first stage (Eqs. 7 and 10) is used.
  * the embedding activation 8sbhp (Eq. 13) is used as printed.
  * the activation terms are for the first pipeline stage (Eq. 16-17), which
    holds L layers of activations under 1F1B.
"""
from fractions import Fraction as Fr


def layer_params(h, a, k, h_ffn, t=1):
    """Parameters of one transformer layer on one TP rank: attention
    2h^2(1+k/a) (Eq. 1) and FFN 3*h*h_ffn (Eq. 2) divided by t (Sec. 3.1.2),
    plus the two replicated RMSNorm gains 2h (Eq. 3)."""
    attn = Fr(2 * h * h * (a + k), a)
    ffn = Fr(3 * h * h_ffn)
    return (attn + ffn) / t + 2 * h


def total_params(h, a, k, h_ffn, L, v):
    """Eq. 3: 2hv + h + L(2h^2(1+k/a) + 3h h_ffn + 2h)."""
    return 2 * h * v + h + L * layer_params(h, a, k, h_ffn)


def params_per_gpu(h, a, k, h_ffn, L, v, t, p):
    """Parameters held by the first pipeline stage of one TP rank."""
    ell = layer_params(h, a, k, h_ffn, t)
    if p == 1:
        return Fr(2 * h * v, t) + h + L * ell
    return Fr(h * v, t) + Fr(L, p) * ell


def act_bytes_per_layer(h, a, k, h_ffn, s, b, t=1, c=1):
    """Eq. 12 divided by t*c (Eqs. 15, 17): sbh(12 + 4k/a + 8h_ffn/h)/(tc)."""
    return Fr(s * b * h, t * c) * (12 + Fr(4 * k, a) + Fr(8 * h_ffn, h))


def act_bytes(h, a, k, h_ffn, L, v, s, b, t, c, p):
    """Eq. 17: sbh/(tc) * ((12 + 4k/a + 8h_ffn/h) L + 8p + [p==1] 4(1+v/h))."""
    per_layer = 12 + Fr(4 * k, a) + Fr(8 * h_ffn, h)
    head = 4 * (1 + Fr(v, h)) if p == 1 else 0
    return Fr(s * b * h, t * c) * (per_layer * L + 8 * p + head)


def estimate(h, a, k, h_ffn, L, v, s, b, t, c, p, n_gpus=None, d=None):
    """Eq. 18 with the p == 1 reading above.  Returns a dict of Fractions:
    params, weight (2 bytes), grad (4), optim (12/(dc)), act, total."""
    if d is None:
        d = Fr(n_gpus, t * c * p)
    psi = params_per_gpu(h, a, k, h_ffn, L, v, t, p)
    out = dict(params=psi, weight=2 * psi, grad=4 * psi, optim=12 * psi / (d * c),
               act_layer=act_bytes_per_layer(h, a, k, h_ffn, s, b, t, c),
               act=act_bytes(h, a, k, h_ffn, L, v, s, b, t, c, p))
    out["total"] = out["weight"] + out["grad"] + out["optim"] + out["act"]
    return out


def gib_2dp(n_bytes):
    """Bytes -> GiB rounded to two decimals, half away from zero (how the
    paper's tables print their estimates)."""
    q = Fr(n_bytes) / (1 << 30) * 100
    n = int(q)
    if q - n >= Fr(1, 2):
        n += 1
    return Fr(n, 100)


def oom_class(total_bytes, device_bytes):
    """The paper's reading of an estimate against the device memory (Sec. 4.1):
    at most 80 % of it -> "green" (trainable: temporary buffers and
    fragmentation fit in the remaining 20 %), at most all of it -> "yellow"
    (may or may not run out of memory), above it -> "red" (out of memory)."""
    if Fr(total_bytes) <= Fr(8, 10) * device_bytes:
        return "green"
    return "yellow" if Fr(total_bytes) <= device_bytes else "red"
