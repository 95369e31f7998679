"""GPU parity of the Adam step over an optimizer shard (l4d_adam_step) against
the oracle (oracle.optim.adam_step, float64).

Every step is compared from the same fp32 state: the oracle steps the arrays
the GPU held before the call.  The bar for the fp32 outputs is derived from
the kernel's arithmetic: each fp32 operation rounds with relative error at
most E = 2^-24, so, with M = beta1 |m| + (1 - beta1) |g| the size of the
momentum sum and u the update direction m_hat / (sqrt(v_hat) + eps),
  |m' - ref| <= 4 E M,     |v' - ref| <= 6 E v'   (a sum of non-negative terms),
  |u' - ref| <= r1 4 E M / denom + 12 E |u|,
  |w' - ref| <= 2 E |w'| + lr (|u' - ref| + 2 E |u|) + 3 E lr wd |w|,
each taken twice over.  The bf16 weight is the decision "nearest bf16 of the
fp32 master as stored", so it must equal the round-to-nearest-even of the
GPU's own master bit for bit; the gradient must be zero where it was cleared
and untouched otherwise; elements past n are never written.
"""
import numpy as np
import pytest
import torch

import paper_2411_06465_amd as L
import workloads as W
from oracle.bf16 import round_bf16, to_bits
from oracle.optim import adam_step

pytestmark = pytest.mark.gpu

E = 2.0 ** -24


def f32(x):
    return float(np.float32(x))


def bounds(g, w0, m0, ref, hp, step):
    """Per-element tolerances of (master, m, v) against the oracle's outputs."""
    w1, m1, v1, _ = ref
    b1, b2 = f32(hp["beta1"]), f32(hp["beta2"])
    lr, eps, wd = f32(hp["lr"]), f32(hp["eps"]), f32(hp["weight_decay"])
    r1 = 1.0 / (1.0 - b1 ** step)
    rs2 = 1.0 / np.sqrt(1.0 - b2 ** step)
    big_m = b1 * np.abs(m0) + (1.0 - b1) * np.abs(g)
    denom = np.sqrt(v1) * rs2 + eps
    u = m1 * r1 / denom
    tol_u = r1 * 4 * E * big_m / denom + 12 * E * np.abs(u)
    tol_w = 2 * E * np.abs(w1) + lr * (tol_u + 2 * E * np.abs(u)) + 3 * E * lr * wd * np.abs(w0)
    return 2 * tol_w, 2 * 4 * E * big_m, 2 * 6 * E * v1


def dev(a, pad=0):
    """fp32 device copy of `a` followed by `pad` guard elements of value 7."""
    t = torch.full((a.size + pad,), 7.0, dtype=torch.float32, device="cuda")
    t[: a.size] = torch.from_numpy(np.ascontiguousarray(a, np.float32))
    return t


def host(t, n):
    return t[:n].double().cpu().numpy()


def run_and_check(name, state, n, step, hp, scale_dev=None, zero_grad=False, pad=16):
    """One l4d_adam_step on the first n elements of `state` (host fp32 arrays),
    checked against the oracle; returns the GPU's new state (host fp32)."""
    print(f"\n[adam {name}] n={n} step={step} hp={hp} scale_dev={scale_dev} zero_grad={zero_grad}", flush=True)
    g, w, m, v = (dev(state[k], pad) for k in ("grad", "master", "m", "v"))
    wb = torch.full((n + pad,), 3, dtype=torch.int16, device="cuda")
    sd = None if scale_dev is None else torch.tensor([scale_dev], dtype=torch.float32, device="cuda")
    L.l4d_adam_step(g, w, m, v, wb, step, n=n, grad_scale_dev=sd, zero_grad=zero_grad, **hp)
    torch.cuda.synchronize()
    scale = f32(hp.get("grad_scale", 1.0)) * (1.0 if scale_dev is None else f32(scale_dev))
    g0 = state["grad"][:n].astype(np.float64)
    ref = adam_step(g0, state["master"][:n], state["m"][:n], state["v"][:n], step,
                    lr=f32(hp["lr"]), beta1=f32(hp["beta1"]), beta2=f32(hp["beta2"]), eps=f32(hp["eps"]),
                    weight_decay=f32(hp.get("weight_decay", 0.0)), grad_scale=scale)
    hw = {**hp, "weight_decay": hp.get("weight_decay", 0.0)}
    tol_w, tol_m, tol_v = bounds(g0 * scale, state["master"][:n].astype(np.float64),
                                 state["m"][:n].astype(np.float64), ref, hw, step)
    got_w, got_m, got_v = host(w, n), host(m, n), host(v, n)
    for nm, got, want, tol in (("master", got_w, ref[0], tol_w), ("m", got_m, ref[1], tol_m),
                               ("v", got_v, ref[2], tol_v)):
        bad = np.abs(got - want) > tol
        assert not bad.any(), (f"{nm}: {int(bad.sum())} of {n} beyond the bound, first at "
                               f"{int(np.argmax(bad))}: got {got[bad][0]!r} want {want[bad][0]!r}")
    bits = wb[:n].cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, to_bits(round_bf16(got_w)), err_msg="bf16 weight != RNE(master)")
    gh = g[:n].cpu().numpy()
    np.testing.assert_array_equal(gh, np.zeros(n, np.float32) if zero_grad else state["grad"][:n])
    for t in (g, w, m, v):
        assert bool((t[n:] == 7.0).all()), "an element past n was written"
    assert bool((wb[n:] == 3).all()), "a weight past n was written"
    return dict(grad=state["grad"], master=w[:n].cpu().numpy(), m=m[:n].cpu().numpy(), v=v[:n].cpu().numpy())


HP = dict(lr=1.5e-4, beta1=0.9, beta2=0.95, eps=1e-5, weight_decay=0.1)


def test_three_steps_from_zero_state_ragged():
    # 5,000,003 parameters: 4883 workgroups, the last one partly idle, and a tail of 3
    n = 5_000_003
    st = W.adam_inputs("adam-ragged", n)
    st["m"][:] = 0.0
    st["v"][:] = 0.0
    for step in (1, 2, 3):
        nxt = run_and_check("ragged", st, n, step, HP)
        st = dict(W.adam_inputs(f"adam-ragged-{step}", n), master=nxt["master"], m=nxt["m"], v=nxt["v"])


def test_mid_training_state_plain_adam():
    n = 1 << 20
    st = W.adam_inputs("adam-mid", n)
    run_and_check("mid", st, n, 1000, dict(HP, weight_decay=0.0, beta2=0.999, eps=1e-8, lr=1e-3))


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 7, 64, 1027, 3073])
def test_small_shards_with_scales_and_cleared_grad(n):
    st = W.adam_inputs(f"adam-small-{n}", n)
    run_and_check(f"small-{n}", st, n, 7, dict(HP, grad_scale=0.5), scale_dev=0.8, zero_grad=True)


def test_sign_descent_corner():
    # beta1 = beta2 = 0, eps = 0, no decay: the step is lr * sign(g) exactly
    n = 4099
    st = W.adam_inputs("adam-sign", n)
    out = run_and_check("sign", st, n, 5, dict(lr=1.0 / 1024, beta1=0.0, beta2=0.0, eps=0.0))
    want = st["master"].astype(np.float32) - np.float32(1.0 / 1024) * np.sign(st["grad"]).astype(np.float32)
    np.testing.assert_array_equal(out["master"], want)


def test_empty_shard_launches_nothing():
    t = torch.full((16,), 7.0, dtype=torch.float32, device="cuda")
    g, w, m, v = t.clone(), t.clone(), t.clone(), t.clone()
    wb = torch.zeros(16, dtype=torch.int16, device="cuda")
    L.l4d_adam_step(g, w, m, v, wb, 1, n=0, **HP)
    torch.cuda.synchronize()
    for x in (g, w, m, v):
        assert bool((x == 7.0).all())
    assert bool((wb == 0).all())


def test_full_size_70b_shard_sampled():
    """The 300,261,376-parameter shard the benchmark steps, in the same launch:
    sampled elements against the oracle, every output finite, the bf16 weight
    the rounding of the master everywhere."""
    w = W.ADAM_70B_SHARD
    print(f"\n[adam full-size {w.name}] n={w.n}", flush=True)
    st = W.adam_inputs_device(w.name, w.n)
    rng = np.random.default_rng(11)
    idx = np.unique(np.concatenate([[0, 1, 2, 3, w.n - 4, w.n - 3, w.n - 2, w.n - 1],
                                    rng.integers(0, w.n, 200_000)]))
    ti = torch.from_numpy(idx).cuda()
    before = {k: st[k][ti].cpu().numpy() for k in ("grad", "master", "m", "v")}
    wb = torch.empty(w.n, dtype=torch.int16, device="cuda")
    hp = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)
    L.l4d_adam_step(st["grad"], st["master"], st["m"], st["v"], wb, w.step, **hp)
    torch.cuda.synchronize()
    for k in ("master", "m", "v"):
        assert bool(torch.isfinite(st[k]).all()), k
    ref = adam_step(before["grad"], before["master"], before["m"], before["v"], w.step,
                    lr=f32(w.lr), beta1=f32(w.beta1), beta2=f32(w.beta2), eps=f32(w.eps),
                    weight_decay=f32(w.weight_decay))
    tol_w, tol_m, tol_v = bounds(before["grad"].astype(np.float64), before["master"].astype(np.float64),
                                 before["m"].astype(np.float64), ref, hp, w.step)
    for k, want, tol in (("master", ref[0], tol_w), ("m", ref[1], tol_m), ("v", ref[2], tol_v)):
        got = st[k][ti].double().cpu().numpy()
        assert not (np.abs(got - want) > tol).any(), k
    # bf16 weight == RNE(master) over the whole shard, in chunks, by integer arithmetic on the bits
    for lo in range(0, w.n, 1 << 26):
        hi = min(w.n, lo + (1 << 26))
        u = st["master"][lo:hi].view(torch.int32).cpu().numpy().view(np.uint32).astype(np.uint64)
        rne = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
        np.testing.assert_array_equal(wb[lo:hi].cpu().numpy().view(np.uint16), rne)
    del st, wb
    torch.cuda.empty_cache()
