"""Oracle: one GPU's share of a Llama decoder layer, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain float64 numpy,
written for reading, not speed: full-matrix softmax attention, one head at a
time, no blocking or fusion.

What is computed (Sec. 3, Fig. "Llama Architecture" as described in the text):
a pre-norm decoder layer without dropout or biases,

    xn1 = RMSNorm(x; g1)                    h1 = x + Attn(xn1) W_O^T
    [Q|K|V] = xn1 [W_Q|W_K|W_V]^T           xn2 = RMSNorm(h1; g2)
    Q, K <- RoPE(Q), RoPE(K)                y = h1 + (silu(G) * U) W_down^T
    Attn = causal GQA softmax(Q K^T / sqrt(d_h)) V,   [G|U] = xn2 [W_gate|W_up]^T

restricted to one tensor-parallel (TP) rank and one context-parallel (CP) rank.
The shard follows the paper's parallel layout: TP divides heads and the FFN
width by t (Sec. 3.1.2), sequence parallelism (SP) divides the norm/residual
rows by t (Sec. 3.2.1), CP divides the sequence by c (Sec. 2.1, Sec. 3.2.3).
Whatever another rank would contribute through a collective is an explicit
input (``peers``) and whatever this rank would send is an explicit output.

Readings of points the paper leaves open:
  * RMSNorm: y = g * x / sqrt(mean(x^2) + eps), statistics per token row.
  * RoPE (not named by the paper, used by Llama): rotate-half pairs (i, i+d/2),
    angle = position * base**(-2i/d), position = global token index.
  * GQA: q-head i of a rank uses kv-head floor(i / (a/k)) of the same rank.
  * causal mask: a query sees keys at global positions <= its own.
  * CP layout: the sequence is cut into 2c equal chunks; CP rank r owns chunks
    r and 2c-1-r (in that order); the other ranks' K and V arrive as
    ``remote_k``/``remote_v`` holding the remaining chunks in increasing order.
  * SP layout: TP rank r owns local rows [r*s_sp, (r+1)*s_sp).  All-gathers
    insert the peers' rows (``sp_peer_*`` with (t-1)*s_sp rows, in rank order
    without the own rank); a reduce-scatter delivers the sum of the peers'
    partial rows for the own rows (``sp_peer_o`` etc., absent = zero).  In the
    backward the CP ring returns the other ranks' dK/dV for the local keys
    (``cp_peer_dk``/``cp_peer_dv``, absent = zero) and this rank's dK/dV for the
    remote keys leave as ``d_remote_k``/``d_remote_v``.
  * SwiGLU: act = silu(G), prod = act * U; the stash keeps G, U, act, prod.
  * storage: every tensor the layer stores is bf16 (Sec. 3.2 counts 2 bytes
    per activation); each stored tensor is computed from the stored values of
    its inputs and rounded once.  In the backward, the gradients that are the
    operands of products (dG|dU, dh1, d ctx, dQ|dK|dV) are stored in bf16 as
    well; d(xn2), d(xn1) and the copy of dh1 that dx adds are kept in fp32
    (they feed only the RMSNorm backward), so they are not rounded here.
    Weight and norm-gain gradients are float32 accumulators in the library
    (Sec. 3.1: gradients accumulate in FP32) and are returned here in float64.
"""
import numpy as np

from .bf16 import round_bf16


class Shard:
    """Shapes of one (TP rank, CP rank) shard; symbols of the paper's Table 1."""

    def __init__(self, hidden, n_heads, n_kv_heads, ffn, seq, micro_batch=1,
                 tp=1, cp=1, tp_rank=0, cp_rank=0, rms_eps=1e-5, rope_base=1e4):
        self.h, self.a, self.k, self.h_ffn = hidden, n_heads, n_kv_heads, ffn
        self.s, self.b, self.t, self.c = seq, micro_batch, tp, cp
        self.tp_rank, self.cp_rank = tp_rank, cp_rank
        self.eps, self.base = rms_eps, rope_base
        self.d_h = hidden // n_heads
        self.a_t, self.k_t, self.f_t = n_heads // tp, n_kv_heads // tp, ffn // tp
        self.group = n_heads // n_kv_heads
        self.s_c = seq // cp
        self.s_sp = self.s_c // tp

    def chunks(self):
        """Global chunk ids owned by this CP rank, and the remote ones."""
        if self.c == 1:
            return [0], []
        own = [self.cp_rank, 2 * self.c - 1 - self.cp_rank]
        return own, [i for i in range(2 * self.c) if i not in own]

    def positions(self):
        """(global positions of local tokens, of remote tokens)."""
        n = self.s // (2 * self.c) if self.c > 1 else self.s
        own, rem = self.chunks()
        span = lambda ids: (np.concatenate([np.arange(i * n, (i + 1) * n) for i in ids])
                            if ids else np.zeros(0, dtype=np.int64))
        return span(own), span(rem)

    def own_rows(self):
        return slice(self.tp_rank * self.s_sp, (self.tp_rank + 1) * self.s_sp)


# ---------------------------------------------------------------- SP collectives

def gather(sh, own, peer):
    """All-gather over the TP group: [b, s_sp, h] own rows + [b, (t-1)s_sp, h]
    peer rows -> [b, s_c, h] in rank order."""
    if sh.t == 1:
        return own
    r, n = sh.tp_rank, sh.s_sp
    return np.concatenate([peer[:, :r * n], own, peer[:, r * n:]], axis=1)


def split_own(sh, full):
    """Inverse of ``gather``: (own rows, peer rows in rank order)."""
    if sh.t == 1:
        return full, full[:, :0]
    r, n = sh.tp_rank, sh.s_sp
    return full[:, r * n:(r + 1) * n], np.concatenate([full[:, :r * n], full[:, (r + 1) * n:]], axis=1)


# ---------------------------------------------------------------- building blocks

def rmsnorm(x, gain, eps):
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * rstd * gain


def rmsnorm_bwd(x, gain, eps, dy):
    """Gradient of rmsnorm w.r.t. x and gain (gain gradient summed over rows)."""
    n = x.shape[-1]
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    xhat = x * rstd
    gdy = gain * dy
    dx = rstd * (gdy - xhat * np.sum(gdy * xhat, axis=-1, keepdims=True) / n)
    dgain = np.sum(dy * xhat, axis=tuple(range(x.ndim - 1)))
    return dx, dgain


def rope(x, pos, d_h, base, inverse=False):
    """Rotate-half RoPE on [b, n, heads*d_h]; ``inverse`` rotates by -angle
    (the transpose, i.e. the backward of the forward rotation)."""
    b, n, w = x.shape
    xs = x.reshape(b, n, w // d_h, d_h)
    half = d_h // 2
    inv_freq = base ** (-2.0 * np.arange(half) / d_h)
    ang = pos[:, None].astype(np.float64) * inv_freq[None, :]          # [n, half]
    if inverse:
        ang = -ang
    cos, sin = np.cos(ang)[None, :, None, :], np.sin(ang)[None, :, None, :]
    x1, x2 = xs[..., :half], xs[..., half:]
    out = np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)
    return out.reshape(b, n, w)


def silu(g):
    return g / (1.0 + np.exp(-g))


def _heads(x, d_h):
    b, n, w = x.shape
    return x.reshape(b, n, w // d_h, d_h)


def attention(sh, Q, K, V, q_pos, k_pos):
    """Causal GQA softmax attention with the full score matrix.
    Q [b, n_q, a_t*d_h]; K, V [b, n_k, k_t*d_h] (local then remote tokens).
    Returns ctx [b, n_q, a_t*d_h] and the row log-sum-exp [b, a_t, n_q]."""
    d, scale = sh.d_h, 1.0 / np.sqrt(sh.d_h)
    q, k, v = _heads(Q, d), _heads(K, d), _heads(V, d)
    visible = k_pos[None, :] <= q_pos[:, None]                           # [n_q, n_k]
    ctx = np.zeros_like(q)
    lse = np.zeros((Q.shape[0], sh.a_t, Q.shape[1]))
    for bi in range(Q.shape[0]):
        for hq in range(sh.a_t):
            hk = hq // sh.group
            s = (q[bi, :, hq] @ k[bi, :, hk].T) * scale
            s = np.where(visible, s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            z = e.sum(axis=1, keepdims=True)
            ctx[bi, :, hq] = (e / z) @ v[bi, :, hk]
            lse[bi, hq] = (m + np.log(z))[:, 0]
    return ctx.reshape(Q.shape), lse


def attention_bwd(sh, Q, K, V, q_pos, k_pos, dctx):
    """Exact gradient of ``attention`` (P recomputed from Q and K, as
    FlashAttention does instead of storing it, Sec. 3.2)."""
    d, scale = sh.d_h, 1.0 / np.sqrt(sh.d_h)
    q, k, v, do = _heads(Q, d), _heads(K, d), _heads(V, d), _heads(dctx, d)
    visible = k_pos[None, :] <= q_pos[:, None]
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    for bi in range(Q.shape[0]):
        for hq in range(sh.a_t):
            hk = hq // sh.group
            s = np.where(visible, (q[bi, :, hq] @ k[bi, :, hk].T) * scale, -np.inf)
            p = np.exp(s - s.max(axis=1, keepdims=True))
            p /= p.sum(axis=1, keepdims=True)
            dp = do[bi, :, hq] @ v[bi, :, hk].T
            ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
            dq[bi, :, hq] = (ds @ k[bi, :, hk]) * scale
            dk[bi, :, hk] += (ds.T @ q[bi, :, hq]) * scale
            dv[bi, :, hk] += p.T @ do[bi, :, hq]
    return dq.reshape(Q.shape), dk.reshape(K.shape), dv.reshape(V.shape)


def _tokens_t(a, b):
    """sum over batch and tokens of a^T b: [b, n, p], [b, n, q] -> [p, q]."""
    return a.reshape(-1, a.shape[-1]).T @ b.reshape(-1, b.shape[-1])


# ---------------------------------------------------------------- the layer

def layer_forward(sh, w, x, peers=None, exact=False):
    """One rank's forward.  ``w``: norm1 [h], qkv [(a_t+2k_t)d_h, h], o [h, a_t d_h],
    norm2 [h], gate_up [2 f_t, h] (gate rows then up rows), down [h, f_t].
    ``x``: the rank's own rows [b, s_sp, h].  Returns a dict with ``y`` and the
    stash (x, xn1, q, k, v, ctx, h1, xn2, gate, up, act, prod), the attention
    ``lse`` and the partial rows sent to peers (``o_send``, ``ffn_send``)."""
    peers = peers or {}
    rnd = (lambda a: a) if exact else round_bf16
    pos, rpos = sh.positions()
    d = sh.d_h
    nq, nk = sh.a_t * d, sh.k_t * d

    xn1 = rnd(rmsnorm(x, w["norm1"], sh.eps))
    qkv = gather(sh, xn1, peers.get("sp_peer_xn1")) @ w["qkv"].T
    q = rnd(rope(qkv[..., :nq], pos, d, sh.base))
    k = rnd(rope(qkv[..., nq:nq + nk], pos, d, sh.base))
    v = rnd(qkv[..., nq + nk:])
    k_all, v_all, k_pos = k, v, pos
    if sh.c > 1:
        k_all = np.concatenate([k, peers["remote_k"]], axis=1)
        v_all = np.concatenate([v, peers["remote_v"]], axis=1)
        k_pos = np.concatenate([pos, rpos])
    ctx_f, lse = attention(sh, q, k_all, v_all, pos, k_pos)
    ctx = rnd(ctx_f)

    o_own, o_peer = split_own(sh, ctx @ w["o"].T)
    h1 = x + o_own
    if peers.get("sp_peer_o") is not None:
        h1 = h1 + peers["sp_peer_o"]
    h1 = rnd(h1)

    xn2 = rnd(rmsnorm(h1, w["norm2"], sh.eps))
    gu = gather(sh, xn2, peers.get("sp_peer_xn2")) @ w["gate_up"].T
    gate, up = rnd(gu[..., :sh.f_t]), rnd(gu[..., sh.f_t:])
    a = silu(gate)
    act, prod = rnd(a), rnd(a * up)

    f_own, f_peer = split_own(sh, prod @ w["down"].T)
    y = h1 + f_own
    if peers.get("sp_peer_ffn") is not None:
        y = y + peers["sp_peer_ffn"]
    y = rnd(y)
    return dict(y=y, x=x, xn1=xn1, q=q, k=k, v=v, ctx=ctx, h1=h1, xn2=xn2,
                gate=gate, up=up, act=act, prod=prod, lse=lse,
                o_send=rnd(o_peer), ffn_send=rnd(f_peer))


def layer_backward(sh, w, st, dy, peers=None, exact=False):
    """One rank's backward from the stash ``st`` of ``layer_forward`` and the own
    rows of the output gradient ``dy`` [b, s_sp, h].  Returns dx, the gradients
    d_<weight> (float64), d_remote_k / d_remote_v (CP), and the partial rows sent
    to peers by the backward reduce-scatters (``dxn2_send``, ``dxn1_send``)."""
    peers = peers or {}
    rnd = (lambda a: a) if exact else round_bf16
    pos, rpos = sh.positions()
    d = sh.d_h
    nq, nk = sh.a_t * d, sh.k_t * d
    out = {}

    # FFN: y = h1 + prod W_down^T, prod = silu(gate) * up
    dy_full = gather(sh, dy, peers.get("sp_peer_dy"))
    out["d_down"] = _tokens_t(dy_full, st["prod"])
    dprod = dy_full @ w["down"]                 # consumed directly, not stored
    sg = 1.0 / (1.0 + np.exp(-st["gate"]))
    dgate = dprod * st["up"] * (sg * (1.0 + st["gate"] * (1.0 - sg)))
    dup = dprod * st["act"]
    dgu = rnd(np.concatenate([dgate, dup], axis=-1))
    xn2_full = gather(sh, st["xn2"], peers.get("sp_peer_xn2"))
    out["d_gate_up"] = _tokens_t(dgu, xn2_full)
    dxn2_own, dxn2_peer = split_own(sh, dgu @ w["gate_up"])
    if peers.get("sp_peer_dxn2") is not None:
        dxn2_own = dxn2_own + peers["sp_peer_dxn2"]
    dxn2 = dxn2_own                             # kept in fp32: feeds only the norm backward
    out["dxn2_send"] = rnd(dxn2_peer)
    dh1_n, out["d_norm2"] = rmsnorm_bwd(st["h1"], w["norm2"], sh.eps, dxn2)
    dh1_res = dy + dh1_n                        # fp32: the residual added into dx
    dh1 = rnd(dh1_res)                          # bf16: operand of the O-projection products

    # attention block: h1 = x + ctx W_O^T
    dh1_full = gather(sh, dh1, peers.get("sp_peer_dh1"))
    out["d_o"] = _tokens_t(dh1_full, st["ctx"])
    dctx = rnd(dh1_full @ w["o"])
    k_all, v_all, k_pos = st["k"], st["v"], pos
    if sh.c > 1:
        k_all = np.concatenate([st["k"], peers["remote_k"]], axis=1)
        v_all = np.concatenate([st["v"], peers["remote_v"]], axis=1)
        k_pos = np.concatenate([pos, rpos])
    dq, dk_all, dv_all = attention_bwd(sh, st["q"], k_all, v_all, pos, k_pos, dctx)
    n_loc = st["k"].shape[1]
    dk_loc, dv_loc = dk_all[:, :n_loc], dv_all[:, :n_loc]
    if peers.get("cp_peer_dk") is not None:     # other CP ranks' share for our keys
        dk_loc = dk_loc + peers["cp_peer_dk"]
        dv_loc = dv_loc + peers["cp_peer_dv"]
    dq = rnd(rope(dq, pos, d, sh.base, inverse=True))
    dk = rnd(rope(dk_loc, pos, d, sh.base, inverse=True))
    dv = rnd(dv_loc)
    if sh.c > 1:
        out["d_remote_k"] = rnd(dk_all[:, n_loc:])
        out["d_remote_v"] = rnd(dv_all[:, n_loc:])
    dqkv = np.concatenate([dq, dk, dv], axis=-1)
    xn1_full = gather(sh, st["xn1"], peers.get("sp_peer_xn1"))
    out["d_qkv"] = _tokens_t(dqkv, xn1_full)
    dxn1_own, dxn1_peer = split_own(sh, dqkv @ w["qkv"])
    if peers.get("sp_peer_dxn1") is not None:
        dxn1_own = dxn1_own + peers["sp_peer_dxn1"]
    dxn1 = dxn1_own                             # kept in fp32: feeds only the norm backward
    out["dxn1_send"] = rnd(dxn1_peer)
    dx_n, out["d_norm1"] = rmsnorm_bwd(st["x"], w["norm1"], sh.eps, dxn1)
    out["dx"] = rnd(dh1_res + dx_n)
    # intermediates, for localising a mismatch
    out.update(dgu=dgu, dxn2=dxn2, dh1=dh1, dctx=dctx, dqkv=dqkv, dxn1=dxn1)
    return out
