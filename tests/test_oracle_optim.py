"""Pins of the oracle's Adam step (Sec. 3.1: BF16 weight, FP32 gradient, FP32
master weight / momentum / variance) against what the algorithm fixes: closed
forms of special cases, the step-size bound, and torch's own implementation of
the same published algorithm (CPU, float64)."""
import numpy as np
import pytest
import torch

from oracle.bf16 import round_bf16
from oracle.optim import adam_step


def rand(n, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(n) * scale


def test_first_step_is_lr_times_g_over_abs_g():
    # from zero moments, bias correction gives m_hat = g, v_hat = g^2
    g, w = rand(1000, 1), rand(1000, 2)
    w1, m1, v1, _ = adam_step(g, w, np.zeros(1000), np.zeros(1000), 1, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)
    np.testing.assert_allclose(w1, w - 1e-3 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-15)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v1, 0.001 * g * g, rtol=1e-12)


def test_zero_betas_give_sign_descent():
    g, w = rand(500, 3), rand(500, 4)
    m0, v0 = rand(500, 5), np.abs(rand(500, 6))
    w1, _, _, _ = adam_step(g, w, m0, v0, 7, lr=0.01, beta1=0.0, beta2=0.0, eps=0.0)
    np.testing.assert_allclose(w1, w - 0.01 * np.sign(g), rtol=0, atol=1e-15)


def test_decay_only_shrinks_the_weight():
    w = rand(300, 7)
    w1, m1, v1, _ = adam_step(np.zeros(300), w, np.zeros(300), np.zeros(300), 3, lr=0.1, beta1=0.9,
                              beta2=0.95, eps=1e-6, weight_decay=0.01)
    np.testing.assert_allclose(w1, w * (1 - 0.1 * 0.01), rtol=1e-15)
    assert not m1.any() and not v1.any()


def test_grad_scale_scales_the_gradient():
    g, w, m, v = rand(200, 8), rand(200, 9), rand(200, 10), np.abs(rand(200, 11))
    a = adam_step(g, w, m, v, 5, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, grad_scale=0.25)
    b = adam_step(0.25 * g, w, m, v, 5, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_step_is_bounded_by_cauchy_schwarz():
    # m_t = (1-b1) sum_k b1^k g_{t-k}, v_t = (1-b2) sum_k b2^k g_{t-k}^2, so by
    # Cauchy-Schwarz |m_hat| / sqrt(v_hat) <= (1-b1)/(1-b1^t) * sqrt((1-b2^t)/(1-b2))
    # * sqrt(sum_{k<t} (b1^2/b2)^k); at t = 1 the bound is 1 and is reached
    rng = np.random.default_rng(12)
    b1, b2, lr = 0.9, 0.99, 1e-2
    w = rng.standard_normal(2000)
    m, v = np.zeros(2000), np.zeros(2000)
    for t in range(1, 40):
        g = rng.standard_normal(2000) * rng.uniform(0.01, 100)
        if t % 7 == 0:
            g = np.abs(g)              # a run of one sign pushes m_hat towards the bound
        w1, m, v, _ = adam_step(g, w, m, v, t, lr=lr, beta1=b1, beta2=b2, eps=0.0)
        bound = ((1 - b1) / (1 - b1 ** t) * np.sqrt((1 - b2 ** t) / (1 - b2))
                 * np.sqrt(sum((b1 * b1 / b2) ** k for k in range(t))))
        step = np.max(np.abs(w1 - w)) / lr
        assert step <= bound * (1 + 1e-12)
        if t == 1:
            assert step == pytest.approx(1.0, rel=1e-12)
        w = w1


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_matches_torch_adamw_over_many_steps(wd):
    n, steps = 4096, 25
    rng = np.random.default_rng(13)
    w0 = rng.standard_normal(n)
    p = torch.nn.Parameter(torch.tensor(w0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=3e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    w, m, v = w0.copy(), np.zeros(n), np.zeros(n)
    for t in range(1, steps + 1):
        g = rng.standard_normal(n) * 0.5
        p.grad = torch.tensor(g)
        opt.step()
        w, m, v, _ = adam_step(g, w, m, v, t, lr=3e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=wd)
    st = opt.state[p]
    np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-18)


def test_weight_is_the_fp32_master_on_the_bf16_grid():
    g, w = rand(1000, 14), rand(1000, 15)
    w1, _, _, wb = adam_step(g, w, np.zeros(1000), np.zeros(1000), 1, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)
    np.testing.assert_array_equal(wb, round_bf16(w1.astype(np.float32).astype(np.float64)))
    assert np.all(np.abs(wb - w1) <= np.abs(w1) * 2.0 ** -8 + 1e-30)


def test_step_counts_from_one():
    with pytest.raises(ValueError):
        adam_step(np.zeros(1), np.zeros(1), np.zeros(1), np.zeros(1), 0, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)


def test_70b_shard_size_is_the_memory_model_share():
    # first pipeline stage of a TP rank of Llama-3-70B at (t, p) = (8, 8), over d c = 4
    import workloads as W
    from oracle.memory import params_per_gpu
    assert W.ADAM_70B_SHARD.n * 4 == params_per_gpu(8192, 64, 8, 28672, 80, 128256, 8, 8)
