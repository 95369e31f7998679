"""Pins of the oracle for the ends of the model (oracle/ends.py): the
vocabulary-parallel embedding and the LM-head block, forward and backward.

Pinned against library routines (torch's embedding, rms_norm, linear and
cross_entropy with autograd, float64), float64 central finite differences,
and shard composition: two TP ranks exchanging their true collective data
reproduce the unsharded result.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ends as E
from oracle.layer import Shard, split_own

RNG = np.random.default_rng(4321)


def shard(t=1, r=0, h=32, s=16, b=2):
    return Shard(hidden=h, n_heads=2, n_kv_heads=1, ffn=64, seq=s, micro_batch=b, tp=t, tp_rank=r)


# ---------------------------------------------------------------- embedding

def test_embedding_single_rank_is_a_table_lookup():
    sh, v = shard(), 50
    w = RNG.standard_normal((v, sh.h))
    ids = RNG.integers(0, v, (sh.b, sh.s_c))
    out = E.embedding_forward(sh, w, ids, 0, exact=True)
    ref = F.embedding(torch.from_numpy(ids), torch.from_numpy(w)).numpy()
    assert np.array_equal(out["own"], ref)


def test_embedding_backward_matches_autograd():
    sh, v = shard(), 20
    w = RNG.standard_normal((v, sh.h))
    ids = RNG.integers(0, v, (sh.b, sh.s_c))          # 64 tokens over 20 rows: repeats
    dy = RNG.standard_normal((sh.b, sh.s_c, sh.h))
    wt = torch.from_numpy(w).requires_grad_()
    F.embedding(torch.from_numpy(ids), wt).backward(torch.from_numpy(dy))
    dw = E.embedding_backward(sh, ids, dy, None, v, 0)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-13, atol=1e-13)


def test_embedding_tensor_parallel_ranks_compose():
    t, v, h = 2, 40, 32
    full = shard(h=h)
    w = RNG.standard_normal((v, h))
    ids = RNG.integers(0, v, (full.b, full.s_c))
    ref = E.embedding_forward(full, w, ids, 0, exact=True)["own"]
    dy_full = RNG.standard_normal((full.b, full.s_c, h))
    dw_ref = E.embedding_backward(full, ids, dy_full, None, v, 0)
    shs = [shard(t=t, r=r, h=h) for r in range(t)]
    v_t = v // t
    outs = [E.embedding_forward(shs[r], w[r * v_t:(r + 1) * v_t], ids, r * v_t, exact=True) for r in range(t)]
    n = shs[0].s_sp
    dws = []
    for r in range(t):
        o = 1 - r
        # the other rank's partial rows for this rank's rows: its send, at this rank's slot
        rows = slice(r * n, (r + 1) * n) if r < o else slice((r - 1) * n, r * n)
        got = E.embedding_forward(shs[r], w[r * v_t:(r + 1) * v_t], ids, r * v_t,
                                  receipt=outs[o]["send"][:, rows], exact=True)["own"]
        assert np.array_equal(got, split_own(shs[r], ref)[0])
        dy_own, dy_peer = split_own(shs[r], dy_full)
        dws.append(E.embedding_backward(shs[r], ids, dy_own, dy_peer, v_t, r * v_t))
    np.testing.assert_allclose(np.concatenate(dws), dw_ref, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- LM-head block

def head_inputs(sh, v, scale=0.3):
    x = RNG.standard_normal((sh.b, sh.s_sp, sh.h))
    gain = 1 + RNG.standard_normal(sh.h) * 0.1
    w = RNG.standard_normal((v, sh.h)) * scale
    tg = RNG.integers(0, v, (sh.b, sh.s_c))
    return x, gain, w, tg


def test_lm_head_block_matches_autograd():
    sh, v, gs = shard(), 37, 0.7
    x, gain, w, tg = head_inputs(sh, v)
    fw = E.lm_head_forward(sh, x, gain, w, tg, 0, exact=True)
    bw = E.lm_head_backward(sh, x, gain, w, tg, 0, fw, grad_scale=gs, exact=True)
    xt, gt, wt = (torch.from_numpy(a).requires_grad_() for a in (x, gain, w))
    xn = F.rms_norm(xt, (sh.h,), gt, eps=sh.eps)
    logits = (xn.reshape(-1, sh.h) @ wt.T)
    loss = F.cross_entropy(logits, torch.from_numpy(tg.reshape(-1)), reduction="none")
    (loss.sum() * gs).backward()
    np.testing.assert_allclose(fw["loss"], loss.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(fw["probs"], torch.softmax(logits, -1).detach().numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(bw["dx"], xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(bw["d_gain"], gt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(bw["d_w"], wt.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_lm_head_block_matches_finite_differences():
    sh, v = shard(h=16, s=4, b=1), 11
    x, gain, w, tg = head_inputs(sh, v)

    def total(x_, g_, w_):
        return E.lm_head_forward(sh, x_, g_, w_, tg, 0, exact=True)["loss"].sum()

    fw = E.lm_head_forward(sh, x, gain, w, tg, 0, exact=True)
    bw = E.lm_head_backward(sh, x, gain, w, tg, 0, fw, exact=True)
    eps = 1e-6
    for name, arr, grad in (("x", x, bw["dx"]), ("gain", gain, bw["d_gain"]), ("w", w, bw["d_w"])):
        d = RNG.standard_normal(arr.shape)
        args = {"x": x, "gain": gain, "w": w}
        hi = dict(args, **{name: arr + eps * d})
        lo = dict(args, **{name: arr - eps * d})
        fd = (total(hi["x"], hi["gain"], hi["w"]) - total(lo["x"], lo["gain"], lo["w"])) / (2 * eps)
        assert abs(fd - np.sum(grad * d)) <= 1e-6 * max(1.0, abs(fd)), name


def test_lm_head_block_tensor_parallel_ranks_compose():
    t, v, h = 2, 30, 32
    full = shard(h=h)
    x_full = RNG.standard_normal((full.b, full.s_c, h))
    gain = 1 + RNG.standard_normal(h) * 0.1
    w = RNG.standard_normal((v, h)) * 0.3
    tg = RNG.integers(0, v, (full.b, full.s_c))
    fw_ref = E.lm_head_forward(full, x_full, gain, w, tg, 0, exact=True)
    bw_ref = E.lm_head_backward(full, x_full, gain, w, tg, 0, fw_ref, grad_scale=0.5, exact=True)
    shs = [shard(t=t, r=r, h=h) for r in range(t)]
    v_t, n = v // t, shs[0].s_sp
    xs = [split_own(shs[r], x_full)[0] for r in range(t)]
    # pass 1: each rank's normed rows and local statistics
    fw0 = [E.lm_head_forward(shs[r], xs[r], gain, w[r * v_t:(r + 1) * v_t], tg, r * v_t,
                             peer_xn=split_own(shs[r], fw_ref["xn"].reshape(full.b, full.s_c, h))[1],
                             peer_lse=np.zeros(full.b * full.s_c), peer_target_logit=np.zeros(full.b * full.s_c),
                             exact=True)
           for r in range(t)]
    local_lse = [np.log(np.exp(f["logits"]).sum(axis=1)) for f in fw0]
    fws, bws = [], []
    for r in range(t):
        o = 1 - r
        lo = tg.reshape(-1) - o * v_t
        zo = np.where((lo >= 0) & (lo < v_t), fw0[o]["logits"][np.arange(lo.size), np.clip(lo, 0, v_t - 1)], 0.0)
        fw = E.lm_head_forward(shs[r], xs[r], gain, w[r * v_t:(r + 1) * v_t], tg, r * v_t,
                               peer_xn=fw0[o]["xn"], peer_lse=local_lse[o], peer_target_logit=zo, exact=True)
        fws.append(fw)
        np.testing.assert_allclose(fw["loss"], fw_ref["loss"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(fws[0]["probs"].sum(1) + fws[1]["probs"].sum(1), 1.0, rtol=1e-12)
    # backward: the peers' partial d(xn) for the own rows come from their sends
    first = [E.lm_head_backward(shs[r], xs[r], gain, w[r * v_t:(r + 1) * v_t], tg, r * v_t, fws[r], 0.5, exact=True)
             for r in range(t)]
    for r in range(t):
        o = 1 - r
        rows = slice(r * n, (r + 1) * n) if r < o else slice((r - 1) * n, r * n)
        bw = E.lm_head_backward(shs[r], xs[r], gain, w[r * v_t:(r + 1) * v_t], tg, r * v_t, fws[r], 0.5,
                                peer_dxn=first[o]["send"][:, rows], exact=True)
        bws.append(bw)
    for r in range(t):
        np.testing.assert_allclose(bws[r]["dx"], split_own(shs[r], bw_ref["dx"])[0], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(bws[0]["d_gain"] + bws[1]["d_gain"], bw_ref["d_gain"], rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(np.concatenate([b["d_w"] for b in bws]), bw_ref["d_w"], rtol=1e-11, atol=1e-13)
