"""Workload shapes and seeded synthetic inputs.

This module is shared by the tests, the smoke check and the benchmark.  It
holds no arithmetic of the method: only shapes, seeds and random draws.  Both
the HIP library and the CPU oracle receive the very same bytes from here.

Recipe (the paper trains on real text with Llama-3.1 weights, neither of
which is needed to exercise the arithmetic): projection weights N(0, 0.02)
bf16; RMSNorm gains 1 + N(0, 0.02) bf16; layer inputs, upstream gradients,
remote K/V chunks and sequence-parallel peer slices N(0, 1) bf16; target ids
uniform over the full vocabulary; peer log-sum-exp N(12.3, 0.1) and peer
target logits N(0, 1.28) in fp32.  Optimizer shards (fp32): master weights
N(0, 0.02); gradients N(0, 1) times 10^U(-4, -2), so their magnitudes span
two decades; momentum 0.3 times such a draw; variance the square of one.  Every tensor has its own stream, derived
from the master seed, the workload name and the tensor name.
"""
import zlib
from dataclasses import dataclass, field, asdict

import numpy as np

SEED = 20241106


@dataclass(frozen=True)
class LayerWorkload:
    """A Llama decoder-layer shard: global model dims plus the 4D layout."""
    name: str
    hidden: int
    n_heads: int
    n_kv_heads: int
    ffn: int
    seq: int
    micro_batch: int = 1
    tp: int = 1
    cp: int = 1
    pp: int = 1
    n_gpus: int = 1
    tp_rank: int = 0
    cp_rank: int = 0
    rms_eps: float = 1e-5
    rope_base: float = 1e4
    n_layers: int = 2
    vocab: int = 1024

    @property
    def dp(self):
        return self.n_gpus // (self.tp * self.cp * self.pp)

    def model(self):
        return dict(hidden=self.hidden, n_heads=self.n_heads, n_kv_heads=self.n_kv_heads,
                    ffn=self.ffn, n_layers=self.n_layers, vocab=self.vocab,
                    rms_eps=self.rms_eps, rope_base=self.rope_base)

    def parallel(self):
        return dict(seq=self.seq, micro_batch=self.micro_batch, tp=self.tp, cp=self.cp,
                    pp=self.pp, dp=self.dp, tp_rank=self.tp_rank, cp_rank=self.cp_rank)

    def shard_kwargs(self):
        return dict(hidden=self.hidden, n_heads=self.n_heads, n_kv_heads=self.n_kv_heads,
                    ffn=self.ffn, seq=self.seq, micro_batch=self.micro_batch, tp=self.tp,
                    cp=self.cp, tp_rank=self.tp_rank, cp_rank=self.cp_rank,
                    rms_eps=self.rms_eps, rope_base=self.rope_base)

    # derived shard sizes (plain bookkeeping)
    @property
    def d_h(self):
        return self.hidden // self.n_heads

    @property
    def s_c(self):
        return self.seq // self.cp

    @property
    def s_sp(self):
        return self.s_c // self.tp

    @property
    def a_t(self):
        return self.n_heads // self.tp

    @property
    def k_t(self):
        return self.n_kv_heads // self.tp

    @property
    def f_t(self):
        return self.ffn // self.tp

    def replace(self, **kw):
        d = asdict(self)
        d.update(kw)
        return LayerWorkload(**d)


@dataclass(frozen=True)
class LMHeadWorkload:
    name: str
    tokens: int
    hidden: int
    vocab: int
    tp: int = 1
    tp_rank: int = 0

    @property
    def v_t(self):
        return self.vocab // self.tp


# The five workloads: a tiny layer, a Llama-2-7B-shaped layer, a Llama-3-8B
# shard at TP2 CP2 (8 GPUs), the Llama-3-8B LM head at TP4 and a Llama-3-70B
# shard at TP8 inside the (TP, CP, PP, MBS) = (8, 1, 8, 1) layout on 256 GPUs.
TINY = LayerWorkload("tiny-h256", 256, 4, 2, 688, 128, rope_base=1e4, n_layers=2, vocab=1024)
LLAMA2_7B = LayerWorkload("llama2-7b-layer", 4096, 32, 32, 11008, 4096, rope_base=1e4,
                          n_layers=32, vocab=32000)
LLAMA3_8B_TP2CP2 = LayerWorkload("llama3-8b-tp2cp2", 4096, 32, 8, 14336, 8192, tp=2, cp=2,
                                 n_gpus=8, rope_base=5e5, n_layers=32, vocab=128256)
LLAMA3_8B_LM_TP4 = LMHeadWorkload("llama3-8b-lmhead-tp4", 8192, 4096, 128256, tp=4)
LLAMA3_70B_TP8 = LayerWorkload("llama3-70b-tp8", 8192, 64, 8, 28672, 8192, tp=8, pp=8,
                               n_gpus=256, rope_base=5e5, n_layers=80, vocab=128256)
LAYER_WORKLOADS = {w.name: w for w in (TINY, LLAMA2_7B, LLAMA3_8B_TP2CP2, LLAMA3_70B_TP8)}


# ---------------------------------------------------------------- random draws

def _rng(*names):
    words = [SEED] + [zlib.crc32(str(n).encode()) for n in names]
    return np.random.default_rng(np.random.SeedSequence(words))


def f32_to_bf16_bits(f):
    """float32 -> bf16 bit pattern, nearest-even (input packing for the draws)."""
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_normal(shape, std=1.0, mean=0.0, *names):
    r = _rng(*names)
    f = r.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        f *= np.float32(std)
    if mean != 0.0:
        f += np.float32(mean)
    return f32_to_bf16_bits(f)


def layer_weights(w: LayerWorkload):
    """bf16 bit arrays of one rank's weight shard (layouts as the library expects)."""
    h, d = w.hidden, w.d_h
    n = w.name
    return dict(
        norm1=bf16_normal((h,), 0.02, 1.0, n, "norm1"),
        qkv=bf16_normal(((w.a_t + 2 * w.k_t) * d, h), 0.02, 0.0, n, "w_qkv"),
        o=bf16_normal((h, w.a_t * d), 0.02, 0.0, n, "w_o"),
        norm2=bf16_normal((h,), 0.02, 1.0, n, "norm2"),
        gate_up=bf16_normal((2 * w.f_t, h), 0.02, 0.0, n, "w_gate_up"),
        down=bf16_normal((h, w.f_t), 0.02, 0.0, n, "w_down"),
    )


def layer_activations(w: LayerWorkload, with_receipts=True):
    """x and dy (own rows) plus every peer input the shard needs."""
    b, h, n = w.micro_batch, w.hidden, w.name
    own = (b, w.s_sp, h)
    out = dict(x=bf16_normal(own, 1.0, 0.0, n, "x"), dy=bf16_normal(own, 1.0, 0.0, n, "dy"))
    peers = {}
    if w.cp > 1:
        kv = (b, w.seq - w.s_c, w.k_t * w.d_h)
        peers["remote_k"] = bf16_normal(kv, 1.0, 0.0, n, "remote_k")
        peers["remote_v"] = bf16_normal(kv, 1.0, 0.0, n, "remote_v")
        if with_receipts:
            loc = (b, w.s_c, w.k_t * w.d_h)
            peers["cp_peer_dk"] = bf16_normal(loc, 0.05, 0.0, n, "cp_peer_dk")
            peers["cp_peer_dv"] = bf16_normal(loc, 0.05, 0.0, n, "cp_peer_dv")
    if w.tp > 1:
        pr = (b, (w.tp - 1) * w.s_sp, h)
        for name in ("sp_peer_xn1", "sp_peer_xn2", "sp_peer_dy", "sp_peer_dh1"):
            peers[name] = bf16_normal(pr, 1.0, 0.0, n, name)
        if with_receipts:
            for name in ("sp_peer_o", "sp_peer_ffn", "sp_peer_dxn2", "sp_peer_dxn1"):
                peers[name] = bf16_normal(own, 1.0, 0.0, n, name)
    out["peers"] = peers
    return out


def lm_head_inputs(w: LMHeadWorkload):
    n = w.name
    out = dict(
        hidden=bf16_normal((w.tokens, w.hidden), 1.0, 0.0, n, "hidden"),
        w_lm=bf16_normal((w.v_t, w.hidden), 0.02, 0.0, n, "w_lm"),
        targets=_rng(n, "targets").integers(0, w.vocab, size=w.tokens, dtype=np.int64),
    )
    if w.tp > 1:
        out["peer_lse"] = (_rng(n, "peer_lse").standard_normal(w.tokens) * 0.1 + 12.3).astype(np.float32)
        out["peer_target_logit"] = (_rng(n, "peer_z").standard_normal(w.tokens) * 1.28).astype(np.float32)
    return out


# ---------------------------------------------------------------- optimizer shards

@dataclass(frozen=True)
class AdamWorkload:
    """One data-parallel rank's shard of the optimizer states: n parameters,
    stepped with the given Adam hyperparameters at step number `step`."""
    name: str
    n: int
    step: int = 1000
    lr: float = 1.5e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-5
    weight_decay: float = 0.1


def _grad_like(r, n):
    g = r.standard_normal(n, dtype=np.float32)
    g *= (10.0 ** r.uniform(-4.0, -2.0, n)).astype(np.float32)
    return g


def adam_inputs(name, n):
    """fp32 arrays grad, master, m, v of n elements for the shard `name`."""
    master = _rng(name, "master").standard_normal(n, dtype=np.float32)
    master *= np.float32(0.02)
    m = _grad_like(_rng(name, "m"), n)
    m *= np.float32(0.3)
    v = _grad_like(_rng(name, "v"), n)
    v *= v
    return dict(grad=_grad_like(_rng(name, "grad"), n), master=master, m=m, v=v)


def adam_inputs_device(name, n, device="cuda"):
    """The same distributions as adam_inputs, drawn on the GPU by torch's
    seeded generator (a different stream of numbers: for shards of hundreds
    of millions of parameters, where host draws would take minutes)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(zlib.crc32(f"{SEED}:{name}".encode()))

    def grad_like():
        g = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
        g *= torch.pow(10.0, torch.rand(n, generator=gen, device=device, dtype=torch.float32) * 2.0 - 4.0)
        return g

    master = torch.randn(n, generator=gen, device=device, dtype=torch.float32) * 0.02
    m = grad_like() * 0.3
    v = grad_like()
    v *= v
    return dict(grad=grad_like(), master=master, m=m, v=v)


# The optimizer shard of one rank of Llama-3-70B at (TP, CP, PP, DP) = (8, 1, 8, 4)
# on 256 GPUs: the parameters of the first pipeline stage of a tensor-parallel
# rank (1,201,045,504: the LM-head shard and 10 layers), divided over the
# d c = 4 ranks that share the optimizer states.
ADAM_70B_SHARD = AdamWorkload("llama3-70b-tp8pp8dp4-optimizer-shard", 300_261_376)


# ---------------------------------------------------------------- the ends of the model

@dataclass(frozen=True)
class EndsWorkload:
    """Embedding and LM-head block of one (TP, CP) rank: model dims, sequence,
    micro-batch and the layout (TP/CP sizes and ranks)."""
    name: str
    hidden: int
    n_heads: int
    n_kv_heads: int
    ffn: int
    vocab: int
    seq: int
    micro_batch: int = 1
    tp: int = 1
    cp: int = 1
    tp_rank: int = 0
    cp_rank: int = 0
    rms_eps: float = 1e-5

    @property
    def s_c(self):
        return self.seq // self.cp

    @property
    def s_sp(self):
        return self.s_c // self.tp

    @property
    def v_t(self):
        return self.vocab // self.tp

    @property
    def tokens(self):
        return self.micro_batch * self.s_c

    def model(self):
        return dict(hidden=self.hidden, n_heads=self.n_heads, n_kv_heads=self.n_kv_heads, ffn=self.ffn,
                    n_layers=1, vocab=self.vocab, rms_eps=self.rms_eps)

    def parallel(self):
        return dict(seq=self.seq, micro_batch=self.micro_batch, tp=self.tp, cp=self.cp, pp=1, dp=1,
                    tp_rank=self.tp_rank, cp_rank=self.cp_rank)


def ends_inputs(w: EndsWorkload):
    """Embedding: table shard N(0, 0.02) bf16; token ids Zipf-distributed over a
    seeded permutation of the vocabulary (natural text repeats a few ids
    often); the peers' partial rows for the own rows (the table row when
    another rank holds the id, else zero); output gradients N(0, 1).
    LM head: x N(0, 1), final-norm gain 1 + N(0, 0.02), head shard N(0, 0.02),
    targets uniform over the vocabulary, the peers' normed rows N(0, 1), peer
    log-sum-exp N(ln((t-1) v_t), 0.1), peer target logits N(0, 1.28), the
    peers' partial d(xn) N(0, 0.02 / tokens)."""
    n, b, h, t = w.name, w.micro_batch, w.hidden, w.tp
    own, peer = (b, w.s_sp, h), (b, (t - 1) * w.s_sp, h)
    perm = _rng(n, "perm").permutation(w.vocab)
    ids = perm[(_rng(n, "zipf").zipf(1.3, size=(b, w.s_c)) - 1) % w.vocab].astype(np.int64)
    v0 = w.tp_rank * w.v_t
    own_ids = ids[:, w.tp_rank * w.s_sp:(w.tp_rank + 1) * w.s_sp]
    elsewhere = (own_ids < v0) | (own_ids >= v0 + w.v_t)
    receipt = _rng(n, "receipt").standard_normal(own, dtype=np.float32) * np.float32(0.02)
    receipt *= elsewhere[..., None]
    out = dict(
        w_emb=bf16_normal((w.v_t, h), 0.02, 0.0, n, "w_emb"), ids=ids, emb_receipt=f32_to_bf16_bits(receipt),
        dx_emb=bf16_normal(own, 1.0, 0.0, n, "dx_emb"),
        x=bf16_normal(own, 1.0, 0.0, n, "x"), w_norm=bf16_normal((h,), 0.02, 1.0, n, "w_norm"),
        w_lm=bf16_normal((w.v_t, h), 0.02, 0.0, n, "w_lm"),
        targets=_rng(n, "targets").integers(0, w.vocab, size=w.tokens, dtype=np.int64),
    )
    if t > 1:
        out["peer_dx_emb"] = bf16_normal(peer, 1.0, 0.0, n, "peer_dx_emb")
        out["peer_xn"] = bf16_normal(peer, 1.0, 0.0, n, "peer_xn")
        out["peer_lse"] = (_rng(n, "peer_lse").standard_normal(w.tokens) * 0.1
                           + np.log((t - 1) * w.v_t)).astype(np.float32)
        out["peer_target_logit"] = (_rng(n, "peer_z").standard_normal(w.tokens) * 1.28).astype(np.float32)
        out["peer_dxn"] = bf16_normal(own, 0.02 / w.tokens, 0.0, n, "peer_dxn")
    return out


ENDS_TINY = EndsWorkload("ends-tiny", 256, 4, 2, 688, 1024, 128)
ENDS_TP2CP2_RAGGED = EndsWorkload("ends-tp2cp2-ragged", 512, 4, 2, 1376, 2000, 400, micro_batch=2, tp=2, cp=2,
                                  tp_rank=1, cp_rank=1)
ENDS_MID = EndsWorkload("ends-mid-tp2", 1024, 8, 8, 2816, 8192, 1024, tp=2, tp_rank=0)
# a vocabulary shard of 1288 (not a multiple of 128): d(xn) is summed over two GEMM kernels
ENDS_RAGGED_VOCAB = EndsWorkload("ends-tp2-vocab1288", 512, 4, 2, 1376, 2576, 256, tp=2, tp_rank=1)
# The Llama-3-8B head at TP4 (8192 tokens, vocabulary shard 32064 of 128256).
ENDS_LLAMA3_8B_TP4 = EndsWorkload("ends-llama3-8b-tp4", 4096, 32, 8, 14336, 128256, 8192, tp=4, tp_rank=1)
