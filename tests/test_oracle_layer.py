"""Pins of the layer and LM-head oracles (CPU only).

The paper prints no numeric layer outputs, so the oracle is pinned by what the
mathematics fixes:
  * library routines for the pieces that have one (torch's bf16 cast,
    rms_norm, silu, scaled_dot_product_attention, cross_entropy + autograd),
  * a complex-number restatement of RoPE,
  * closed forms (equal keys -> prefix means, W = 0 -> loss = ln v),
  * float64 central finite differences of <y, dy> on tiny shards (t = 1,
    c = 1 and c = 2 with the remote K/V as inputs; t = 2 with the sends and
    the peers' gradient receipts in the loss),
  * invariants (causality of dx and of dK/dV, RoPE norm preservation),
  * special cases (W_O = W_down = 0 gives y = x and dx = dy bit-exactly),
  * shard composition: t TP ranks, or c CP ranks, exchanging their true
    collective data reproduce the unsharded layer.
"""
import numpy as np
import pytest
import torch

from oracle import layer as Lr
from oracle import lm_head as LM
from oracle.bf16 import round_bf16, from_bits, to_bits

RNG = np.random.default_rng(1234)


def randn(*shape, scale=1.0):
    return RNG.standard_normal(shape) * scale


# ---------------------------------------------------------------- primitives

def test_round_bf16_matches_torch_cast():
    f = (RNG.standard_normal(200_000) * np.exp(RNG.uniform(-30, 30, 200_000))).astype(np.float32)
    ours = round_bf16(f.astype(np.float64))
    ref = torch.from_numpy(f).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


def test_round_bf16_ties_to_even_and_bits_roundtrip():
    one = 1.0
    assert round_bf16(one + 2.0 ** -8) == one                 # tie -> even mantissa
    assert round_bf16(one + 3 * 2.0 ** -8) == one + 2.0 ** -6  # tie -> even mantissa
    assert round_bf16(one + 2.0 ** -8 + 2.0 ** -30) == one + 2.0 ** -7
    x = round_bf16(randn(1000))
    assert np.array_equal(from_bits(to_bits(x)), x)


def test_rmsnorm_matches_torch():
    x, g = randn(3, 5, 64), 1 + randn(64, scale=0.1)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=1e-5)
    assert np.allclose(Lr.rmsnorm(x, g, 1e-5), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_rmsnorm_bwd_matches_autograd():
    x, g, dy = randn(2, 7, 48), 1 + randn(48, scale=0.1), randn(2, 7, 48)
    xt = torch.from_numpy(x).requires_grad_()
    gt = torch.from_numpy(g).requires_grad_()
    torch.nn.functional.rms_norm(xt, (48,), gt, eps=1e-5).backward(torch.from_numpy(dy))
    dx, dg = Lr.rmsnorm_bwd(x, g, 1e-5, dy)
    assert np.allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(dg, gt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_silu_matches_torch():
    g = randn(1000, scale=4)
    assert np.allclose(Lr.silu(g), torch.nn.functional.silu(torch.from_numpy(g)).numpy(), rtol=1e-14)


def test_rope_is_complex_multiplication():
    d_h, base = 16, 500000.0
    x = randn(2, 9, 3 * d_h)
    pos = np.array([0, 1, 2, 7, 100, 2047, 4096, 6000, 8191])
    out = Lr.rope(x, pos, d_h, base)
    xs = x.reshape(2, 9, 3, d_h)
    z = xs[..., :d_h // 2] + 1j * xs[..., d_h // 2:]
    theta = pos[:, None] * base ** (-np.arange(d_h // 2) * 2.0 / d_h)
    zr = z * np.exp(1j * theta)[None, :, None, :]
    ref = np.concatenate([zr.real, zr.imag], axis=-1).reshape(x.shape)
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
    # identity at position 0, norm of every pair preserved, inverse undoes it
    assert np.array_equal(out[:, 0], x[:, 0])
    pairs = lambda a: np.hypot(a.reshape(2, 9, 3, d_h)[..., :d_h // 2], a.reshape(2, 9, 3, d_h)[..., d_h // 2:])
    assert np.allclose(pairs(out), pairs(x), rtol=1e-13)
    assert np.allclose(Lr.rope(out, pos, d_h, base, inverse=True), x, rtol=1e-12, atol=1e-12)


def test_attention_matches_torch_sdpa_gqa():
    sh = Lr.Shard(hidden=64, n_heads=8, n_kv_heads=2, ffn=32, seq=24, micro_batch=2)
    q, k, v = randn(2, 24, 64), randn(2, 24, 16), randn(2, 24, 16)
    pos = np.arange(24)
    ctx, lse = Lr.attention(sh, q, k, v, pos, pos)
    tq = torch.from_numpy(q).view(2, 24, 8, 8).transpose(1, 2)
    tk = torch.from_numpy(k).view(2, 24, 2, 8).transpose(1, 2).repeat_interleave(4, dim=1)
    tv = torch.from_numpy(v).view(2, 24, 2, 8).transpose(1, 2).repeat_interleave(4, dim=1)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    assert np.allclose(ctx, ref.transpose(1, 2).reshape(2, 24, 64).numpy(), rtol=1e-12, atol=1e-12)


def test_attention_equal_keys_gives_prefix_means():
    sh = Lr.Shard(hidden=32, n_heads=2, n_kv_heads=1, ffn=8, seq=10)
    q, v = randn(1, 10, 32), randn(1, 10, 16)
    k = np.repeat(randn(1, 1, 16), 10, axis=1)          # every key identical
    pos = np.arange(10)
    ctx, lse = Lr.attention(sh, q, k, v, pos, pos)
    means = np.cumsum(v[0], axis=0) / np.arange(1, 11)[:, None]
    for hq in range(2):
        assert np.allclose(ctx[0, :, hq * 16:(hq + 1) * 16], means, rtol=1e-12, atol=1e-12)
    # zero queries: every visible score is 0, so lse_i = ln(i + 1)
    _, lse0 = Lr.attention(sh, np.zeros_like(q), k, v, pos, pos)
    assert np.allclose(lse0[0, 0], np.log(np.arange(1, 11)), rtol=1e-14)


def test_attention_bwd_matches_autograd():
    sh = Lr.Shard(hidden=32, n_heads=4, n_kv_heads=2, ffn=8, seq=12)
    q, k, v, do = randn(1, 12, 32), randn(1, 12, 16), randn(1, 12, 16), randn(1, 12, 32)
    pos = np.arange(12)
    dq, dk, dv = Lr.attention_bwd(sh, q, k, v, pos, pos, do)
    tq, tk, tv = (torch.from_numpy(a).requires_grad_() for a in (q, k, v))
    qq = tq.view(1, 12, 4, 8).transpose(1, 2)
    kk = tk.view(1, 12, 2, 8).transpose(1, 2).repeat_interleave(2, dim=1)
    vv = tv.view(1, 12, 2, 8).transpose(1, 2).repeat_interleave(2, dim=1)
    out = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, is_causal=True)
    out.transpose(1, 2).reshape(1, 12, 32).backward(torch.from_numpy(do))
    for ours, ref in ((dq, tq), (dk, tk), (dv, tv)):
        assert np.allclose(ours, ref.grad.numpy(), rtol=1e-11, atol=1e-11)


# ---------------------------------------------------------------- whole layer

def small_shard(**kw):
    base = dict(hidden=32, n_heads=4, n_kv_heads=2, ffn=24, seq=16, rms_eps=1e-5, rope_base=10000.0)
    base.update(kw)
    return Lr.Shard(**base)


def make_weights(sh, scale=0.3):
    d = sh.d_h
    return dict(norm1=1 + randn(sh.h, scale=0.2), qkv=randn((sh.a_t + 2 * sh.k_t) * d, sh.h, scale=scale),
                o=randn(sh.h, sh.a_t * d, scale=scale), norm2=1 + randn(sh.h, scale=0.2),
                gate_up=randn(2 * sh.f_t, sh.h, scale=scale), down=randn(sh.h, sh.f_t, scale=scale))


def make_peers(sh):
    p = {}
    if sh.c > 1:
        p["remote_k"] = randn(sh.b, sh.s - sh.s_c, sh.k_t * sh.d_h)
        p["remote_v"] = randn(sh.b, sh.s - sh.s_c, sh.k_t * sh.d_h)
    return p


def loss_of(sh, w, x, peers, dy):
    return float(np.sum(Lr.layer_forward(sh, w, x, peers, exact=True)["y"] * dy))


@pytest.mark.parametrize("cp", [1, 2])
def test_layer_gradients_match_finite_differences(cp):
    sh = small_shard(cp=cp, micro_batch=2)
    w = make_weights(sh)
    x, dy = randn(sh.b, sh.s_sp, sh.h), randn(sh.b, sh.s_sp, sh.h)
    peers = make_peers(sh)
    st = Lr.layer_forward(sh, w, x, peers, exact=True)
    g = Lr.layer_backward(sh, w, st, dy, peers, exact=True)
    grads = {"x": g["dx"], **{n: g["d_" + n] for n in w}}
    if cp > 1:
        grads["remote_k"], grads["remote_v"] = g["d_remote_k"], g["d_remote_v"]
    eps = 1e-5
    for name, grad in grads.items():
        for _ in range(2):
            def at(sign, direction):
                w2, x2, p2 = dict(w), x, dict(peers)
                if name == "x":
                    x2 = x + sign * eps * direction
                elif name in w:
                    w2[name] = w[name] + sign * eps * direction
                else:
                    p2[name] = peers[name] + sign * eps * direction
                return loss_of(sh, w2, x2, p2, dy)
            direction = randn(*grad.shape)
            fd = (at(1, direction) - at(-1, direction)) / (2 * eps)
            an = float(np.sum(grad * direction))
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


@pytest.mark.parametrize("cp", [1, 2])
def test_tensor_parallel_rank_gradients_match_finite_differences(cp):
    # One TP rank (t = 2, rank 1) with its collective data as fixed inputs.  The
    # backward's peer inputs are the gradients of what this rank hands to the
    # others, so it differentiates
    #   L = <y, dy> + <ffn_send, sp_peer_dy> + <o_send, sp_peer_dh1>
    #       + <xn2, sp_peer_dxn2> + <xn1, sp_peer_dxn1>
    # (the sends feed the peers' y and h1 rows; the receipts are the peers'
    # partial gradients of this rank's normed rows).
    sh = small_shard(tp=2, tp_rank=1, cp=cp, micro_batch=2)
    w = make_weights(sh)
    n_peer = (sh.t - 1) * sh.s_sp
    x, dy = randn(sh.b, sh.s_sp, sh.h), randn(sh.b, sh.s_sp, sh.h)
    peers = make_peers(sh)
    for name in ("sp_peer_xn1", "sp_peer_xn2", "sp_peer_dy", "sp_peer_dh1"):
        peers[name] = randn(sh.b, n_peer, sh.h)
    for name in ("sp_peer_o", "sp_peer_ffn", "sp_peer_dxn2", "sp_peer_dxn1"):
        peers[name] = randn(sh.b, sh.s_sp, sh.h)

    def loss(w2, x2, p2):
        f = Lr.layer_forward(sh, w2, x2, p2, exact=True)
        return float(np.sum(f["y"] * dy) + np.sum(f["ffn_send"] * p2["sp_peer_dy"])
                     + np.sum(f["o_send"] * p2["sp_peer_dh1"]) + np.sum(f["xn2"] * p2["sp_peer_dxn2"])
                     + np.sum(f["xn1"] * p2["sp_peer_dxn1"]))

    st = Lr.layer_forward(sh, w, x, peers, exact=True)
    g = Lr.layer_backward(sh, w, st, dy, peers, exact=True)
    grads = {"x": g["dx"], **{n: g["d_" + n] for n in w}}
    if cp > 1:
        grads["remote_k"], grads["remote_v"] = g["d_remote_k"], g["d_remote_v"]
    eps = 1e-5
    for name, grad in grads.items():
        direction = randn(*grad.shape)

        def at(sign):
            w2, x2, p2 = dict(w), x, dict(peers)
            if name == "x":
                x2 = x + sign * eps * direction
            elif name in w:
                w2[name] = w[name] + sign * eps * direction
            else:
                p2[name] = peers[name] + sign * eps * direction
            return loss(w2, x2, p2)
        fd = (at(1) - at(-1)) / (2 * eps)
        an = float(np.sum(grad * direction))
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_future_keys_get_no_key_or_value_gradient():
    # dy only in row i: K and V of every key after position i receive exactly 0
    sh = small_shard(seq=16)
    w = make_weights(sh)
    x = round_bf16(randn(1, 16, sh.h))
    dy = np.zeros((1, 16, sh.h))
    i = 6
    dy[0, i] = round_bf16(randn(sh.h))
    st = Lr.layer_forward(sh, w, x)
    g = Lr.layer_backward(sh, w, st, dy)
    nq, nk = sh.a_t * sh.d_h, sh.k_t * sh.d_h
    dk, dv = g["dqkv"][0, :, nq:nq + nk], g["dqkv"][0, :, nq + nk:]
    assert np.all(dk[i + 1:] == 0.0) and np.all(dv[i + 1:] == 0.0)
    assert np.any(dk[:i + 1] != 0.0) and np.any(dv[:i + 1] != 0.0)


def test_gradient_is_causal():
    sh = small_shard(seq=16)
    w = make_weights(sh)
    x = round_bf16(randn(1, 16, sh.h))
    dy = np.zeros((1, 16, sh.h))
    i = 6
    dy[0, i] = round_bf16(randn(sh.h))
    st = Lr.layer_forward(sh, w, x)
    g = Lr.layer_backward(sh, w, st, dy)
    assert np.all(g["dx"][0, i + 1:] == 0.0)
    assert np.any(g["dx"][0, :i + 1] != 0.0)


def test_zero_output_projections_give_identity():
    sh = small_shard(cp=2, micro_batch=2)
    w = {n: round_bf16(v) for n, v in make_weights(sh).items()}
    w["o"][:] = 0.0
    w["down"][:] = 0.0
    x = round_bf16(randn(sh.b, sh.s_sp, sh.h))
    dy = round_bf16(randn(sh.b, sh.s_sp, sh.h))
    peers = {n: round_bf16(v) for n, v in make_peers(sh).items()}
    st = Lr.layer_forward(sh, w, x, peers)
    assert np.array_equal(st["y"], x)
    g = Lr.layer_backward(sh, w, st, dy, peers)
    assert np.array_equal(g["dx"], dy)
    assert np.all(g["d_remote_k"] == 0) and np.all(g["d_remote_v"] == 0)


# ---------------------------------------------------------------- shard composition

def tp_slice(sh_full, w, t, r):
    d, a_t, k_t, f_t = sh_full.d_h, sh_full.a // t, sh_full.k // t, sh_full.h_ffn // t
    a, k, f = sh_full.a, sh_full.k, sh_full.h_ffn
    rows = np.concatenate([np.arange(r * a_t * d, (r + 1) * a_t * d),
                           a * d + np.arange(r * k_t * d, (r + 1) * k_t * d),
                           (a + k) * d + np.arange(r * k_t * d, (r + 1) * k_t * d)])
    gu = np.concatenate([np.arange(r * f_t, (r + 1) * f_t), f + np.arange(r * f_t, (r + 1) * f_t)])
    return dict(norm1=w["norm1"], norm2=w["norm2"], qkv=w["qkv"][rows],
                o=w["o"][:, r * a_t * d:(r + 1) * a_t * d], gate_up=w["gate_up"][gu],
                down=w["down"][:, r * f_t:(r + 1) * f_t]), rows, gu


def _peer_rows(sends, t, r, n):
    """Sum over ranks q != r of the rows of q's send buffer destined for r."""
    tot = 0.0
    for q in range(t):
        if q != r:
            idx = r if r < q else r - 1
            tot = tot + sends[q][:, idx * n:(idx + 1) * n]
    return tot


def test_tensor_parallel_ranks_compose_to_unsharded_layer():
    t = 2
    full = small_shard(n_heads=4, n_kv_heads=2, ffn=24, seq=16, micro_batch=2)
    w = make_weights(full)
    x, dy = randn(2, 16, full.h), randn(2, 16, full.h)
    ref_f = Lr.layer_forward(full, w, x, exact=True)
    ref_b = Lr.layer_backward(full, w, ref_f, dy, exact=True)

    shards = [small_shard(n_heads=4, n_kv_heads=2, ffn=24, seq=16, micro_batch=2, tp=t, tp_rank=r)
              for r in range(t)]
    n = shards[0].s_sp
    ws = [tp_slice(full, w, t, r) for r in range(t)]
    xs = [x[:, r * n:(r + 1) * n] for r in range(t)]
    dys = [dy[:, r * n:(r + 1) * n] for r in range(t)]
    others = lambda arrs, r: np.concatenate([arrs[q] for q in range(t) if q != r], axis=1)
    zero_peer = np.zeros((2, (t - 1) * n, full.h))
    peers = [dict(sp_peer_xn1=zero_peer, sp_peer_xn2=zero_peer, sp_peer_dy=others(dys, r),
                  sp_peer_dh1=zero_peer) for r in range(t)]
    for _ in range(6):       # each pass makes one more exchanged quantity correct
        fw = [Lr.layer_forward(shards[r], ws[r][0], xs[r], peers[r], exact=True) for r in range(t)]
        for r in range(t):
            peers[r].update(sp_peer_xn1=others([f["xn1"] for f in fw], r),
                            sp_peer_xn2=others([f["xn2"] for f in fw], r),
                            sp_peer_o=_peer_rows([f["o_send"] for f in fw], t, r, n),
                            sp_peer_ffn=_peer_rows([f["ffn_send"] for f in fw], t, r, n))
    for _ in range(6):
        bw = [Lr.layer_backward(shards[r], ws[r][0], fw[r], dys[r], peers[r], exact=True) for r in range(t)]
        for r in range(t):
            peers[r].update(sp_peer_dh1=others([b["dh1"] for b in bw], r),
                            sp_peer_dxn2=_peer_rows([b["dxn2_send"] for b in bw], t, r, n),
                            sp_peer_dxn1=_peer_rows([b["dxn1_send"] for b in bw], t, r, n))
    close = lambda a, b: np.allclose(a, b, rtol=1e-10, atol=1e-10)
    assert close(np.concatenate([f["y"] for f in fw], axis=1), ref_f["y"])
    assert close(np.concatenate([b["dx"] for b in bw], axis=1), ref_b["dx"])
    for r in range(t):
        _, rows, gu = ws[r]
        d, a_t, f_t = full.d_h, full.a // t, full.h_ffn // t
        assert close(bw[r]["d_qkv"], ref_b["d_qkv"][rows])
        assert close(bw[r]["d_gate_up"], ref_b["d_gate_up"][gu])
        assert close(bw[r]["d_o"], ref_b["d_o"][:, r * a_t * d:(r + 1) * a_t * d])
        assert close(bw[r]["d_down"], ref_b["d_down"][:, r * f_t:(r + 1) * f_t])
    assert close(sum(b["d_norm1"] for b in bw), ref_b["d_norm1"])
    assert close(sum(b["d_norm2"] for b in bw), ref_b["d_norm2"])


def test_context_parallel_ranks_compose_to_unsharded_layer():
    c, s = 2, 16
    full = small_shard(seq=s, micro_batch=2)
    w = make_weights(full)
    x, dy = randn(2, s, full.h), randn(2, s, full.h)
    ref_f = Lr.layer_forward(full, w, x, exact=True)
    ref_b = Lr.layer_backward(full, w, ref_f, dy, exact=True)

    shards = [small_shard(seq=s, micro_batch=2, cp=c, cp_rank=r) for r in range(c)]
    pos = [sh.positions() for sh in shards]
    nl, nr = shards[0].s_c, s - shards[0].s_c
    kvw = full.k_t * full.d_h
    peers = [dict(remote_k=np.zeros((2, nr, kvw)), remote_v=np.zeros((2, nr, kvw))) for _ in range(c)]
    where = {}                 # global position -> (rank, local row)
    for r in range(c):
        for i, p in enumerate(pos[r][0]):
            where[int(p)] = (r, i)

    def remote_of(key, outs, r):
        return np.stack([outs[where[int(p)][0]][key][:, where[int(p)][1]] for p in pos[r][1]], axis=1)

    for _ in range(3):
        fw = [Lr.layer_forward(shards[r], w, x[:, pos[r][0]], peers[r], exact=True) for r in range(c)]
        for r in range(c):
            peers[r]["remote_k"] = remote_of("k", fw, r)
            peers[r]["remote_v"] = remote_of("v", fw, r)
    for r in range(c):
        peers[r]["cp_peer_dk"] = np.zeros((2, nl, kvw))
        peers[r]["cp_peer_dv"] = np.zeros((2, nl, kvw))
    for _ in range(3):
        bw = [Lr.layer_backward(shards[r], w, fw[r], dy[:, pos[r][0]], peers[r], exact=True) for r in range(c)]
        for r in range(c):       # sum what the other ranks computed for r's keys
            dk, dv = np.zeros((2, nl, kvw)), np.zeros((2, nl, kvw))
            for q in range(c):
                if q == r:
                    continue
                for j, p in enumerate(pos[q][1]):
                    owner, row = where[int(p)]
                    if owner == r:
                        dk[:, row] += bw[q]["d_remote_k"][:, j]
                        dv[:, row] += bw[q]["d_remote_v"][:, j]
            peers[r]["cp_peer_dk"], peers[r]["cp_peer_dv"] = dk, dv
    close = lambda a, b: np.allclose(a, b, rtol=1e-10, atol=1e-10)
    for r in range(c):
        assert close(fw[r]["y"], ref_f["y"][:, pos[r][0]])
        assert close(bw[r]["dx"], ref_b["dx"][:, pos[r][0]])
    for name in ("d_qkv", "d_o", "d_gate_up", "d_down", "d_norm1", "d_norm2"):
        assert close(sum(b[name] for b in bw), ref_b[name]), name


@pytest.mark.parametrize("c", [2, 4, 8])
def test_context_parallel_layout_is_a_balanced_partition(c):
    # The CP chunking is meant to balance causal work over ranks: every
    # position is owned once and every rank sees the same number of
    # unmasked (query, key) pairs.
    s = 16 * c
    shards = [small_shard(seq=s, cp=c, cp_rank=r) for r in range(c)]
    owned = np.concatenate([sh.positions()[0] for sh in shards])
    assert np.array_equal(np.sort(owned), np.arange(s))
    for sh in shards:
        loc, rem = sh.positions()
        assert np.array_equal(np.sort(np.concatenate([loc, rem])), np.arange(s))
        assert np.all(np.diff(rem) > 0)
    work = [int(np.sum(np.arange(s)[None, :] <= sh.positions()[0][:, None])) for sh in shards]
    assert len(set(work)) == 1, work


# ---------------------------------------------------------------- LM head

def test_lm_head_zero_weight_gives_ln_v():
    n, h, v, t = 8, 16, 96, 4
    v_t = v // t
    hid = round_bf16(randn(n, h))
    tg = RNG.integers(0, v, n)
    peer_lse = np.full(n, np.log(v - v_t))
    out = LM.lm_head_xent(hid, np.zeros((v_t, h)), tg, 0, peer_lse, np.zeros(n), 1.0 / n, exact=True)
    assert np.allclose(out["loss"], np.log(v), rtol=1e-15)
    onehot = np.zeros((n, v_t))
    own = tg < v_t
    onehot[np.arange(n)[own], tg[own]] = 1.0
    assert np.allclose(out["dlogits"], (1.0 / v - onehot) / n, rtol=1e-14, atol=1e-18)


def test_lm_head_single_shard_matches_torch_cross_entropy():
    n, h, v = 12, 16, 40
    hid, wl = randn(n, h), randn(v, h, scale=0.5)
    tg = RNG.integers(0, v, n)
    out = LM.lm_head_xent(hid, wl, tg, grad_scale=1.0 / n, exact=True)
    th, tw = torch.from_numpy(hid).requires_grad_(), torch.from_numpy(wl).requires_grad_()
    logits = th @ tw.T
    loss = torch.nn.functional.cross_entropy(logits, torch.from_numpy(tg), reduction="none")
    loss.mean().backward()
    assert np.allclose(out["loss"], loss.detach().numpy(), rtol=1e-12)
    assert np.allclose(out["d_hidden"], th.grad.numpy(), rtol=1e-11, atol=1e-14)
    assert np.allclose(out["d_w"], tw.grad.numpy(), rtol=1e-11, atol=1e-14)


def test_lm_head_vocab_parallel_composes():
    n, h, v, t = 10, 16, 64, 4
    v_t = v // t
    hid, wl = randn(n, h), randn(v, h, scale=0.5)
    tg = RNG.integers(0, v, n)
    ref = LM.lm_head_xent(hid, wl, tg, grad_scale=1.0 / n, exact=True)
    logits = hid @ wl.T
    local_lse = [np.log(np.exp(logits[:, r * v_t:(r + 1) * v_t]).sum(1)) for r in range(t)]
    outs = []
    for r in range(t):
        peer = np.logaddexp.reduce([local_lse[q] for q in range(t) if q != r], axis=0)
        z = logits[np.arange(n), tg]
        outs.append(LM.lm_head_xent(hid, wl[r * v_t:(r + 1) * v_t], tg, r * v_t, peer, z, 1.0 / n, exact=True))
    for o in outs:
        assert np.allclose(o["loss"], ref["loss"], rtol=1e-12)
    assert np.allclose(sum(o["d_hidden"] for o in outs), ref["d_hidden"], rtol=1e-11, atol=1e-14)
    assert np.allclose(np.concatenate([o["d_w"] for o in outs]), ref["d_w"], rtol=1e-11, atol=1e-14)
