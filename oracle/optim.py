"""One Adam step over a shard of the 18-bytes-per-parameter layout (Sec. 3.1).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper trains with Adam (it cites Kingma and Ba) in BF16/FP32 mixed
precision: the weight the layers read is BF16, the accumulated gradient FP32,
and the optimizer keeps an FP32 master weight, the gradient momentum and the
gradient variance, sharded over the d*c data- and context-parallel processes
(ZeRO stage 1 / the distributed optimizer).  It gives no hyperparameters.
Readings:
  * the update is Adam's bias-corrected step: with g the (scaled) gradient,
      m <- b1 m + (1 - b1) g,   v <- b2 v + (1 - b2) g^2,
      m_hat = m / (1 - b1^t),   v_hat = v / (1 - b2^t),
      w <- w - lr (m_hat / (sqrt(v_hat) + eps) + wd w)
    with the weight decay decoupled from the gradient (wd = 0 is plain Adam);
  * `grad_scale` multiplies the gradient first (a clipping coefficient the
    caller computed from the global gradient norm; 1 for none);
  * the BF16 weight is the FP32 master weight, as stored, rounded to nearest-even.
Computed in float64 from float64 copies of the inputs.
"""
import numpy as np

from .bf16 import round_bf16


def adam_step(grad, master, m, v, step, lr, beta1, beta2, eps, weight_decay=0.0, grad_scale=1.0):
    """Returns (master, m, v, weight) after step number `step` (1-based); the
    inputs are left unchanged.  weight holds bf16 values as float64."""
    if step < 1:
        raise ValueError("step counts from 1")
    g = np.asarray(grad, np.float64) * grad_scale
    w = np.asarray(master, np.float64)
    m1 = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v1 = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    m_hat = m1 / (1.0 - beta1 ** step)
    v_hat = v1 / (1.0 - beta2 ** step)
    w1 = w - lr * (m_hat / (np.sqrt(v_hat) + eps) + weight_decay * w)
    return w1, m1, v1, round_bf16(w1.astype(np.float32).astype(np.float64))
