"""GPU parity at the full shard sizes the benchmark runs (the Llama-2-7B layer,
the Llama-3-8B TP2 CP2 and Llama-3-70B TP8 layer shards, the Llama-3-8B TP4 LM
head), in the same launch configuration as bench.py.

The full oracle would take too long at these sizes, so the oracle computes
sampled outputs one by one (oracle.layer.layer_forward_rows: K and V for
every token, everything else at the sampled rows; layer_backward_last_rows:
dx at the last local rows, whose backward depends on no other local row;
the LM head per token).  Bar as elsewhere: bf16 outputs within 2e-2 plus one
bf16 step of the oracle value, relative Frobenius 5e-3; the stash byte count
equals Eq. 12 / (tc) exactly.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import layer as OL
from oracle import lm_head as OLM
from oracle import memory as OM
from oracle.bf16 import from_bits
from gpu_common import Buffers, check, host_f64
from test_gpu_lm_head import run_lm

pytestmark = pytest.mark.gpu

LAYERS = [W.LLAMA2_7B, W.LLAMA3_8B_TP2CP2, W.LLAMA3_70B_TP8]


def sample_rows(n, k=6, seed=7):
    """First and last row plus k - 2 seeded others, sorted."""
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, n - 1], rng.choice(np.arange(1, n - 1), k - 2, replace=False)]))


def host_inputs(buf):
    w = buf.w
    sh = OL.Shard(**w.shard_kwargs())
    wts = {k: from_bits(v) for k, v in buf.wbits.items()}
    peers = {k: from_bits(v) for k, v in buf.abits["peers"].items()}
    return sh, wts, from_bits(buf.abits["x"]), from_bits(buf.abits["dy"]), peers


@pytest.mark.parametrize("w", LAYERS, ids=lambda w: w.name)
def test_full_size_layer_forward_at_sampled_rows(w):
    print(f"\n[full-size forward {w.name}] h={w.hidden} heads={w.a_t}/{w.k_t} f_t={w.f_t} s_c={w.s_c} "
          f"tp={w.tp} cp={w.cp}", flush=True)
    buf = Buffers(w)
    saved = buf.run(keep_stash=True)
    assert saved["_bytes"]["formula"] == OM.act_bytes_per_layer(
        w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.seq, w.micro_batch, w.tp, w.cp)
    sh, wts, x, _, peers = host_inputs(buf)
    rows = sample_rows(w.s_sp)
    m = w.tp_rank * w.s_sp + rows
    ref = OL.layer_forward_rows(sh, wts, x, rows, peers)
    rep, ok = [], True
    ok &= check("y", host_f64(buf.y)[:, rows], ref["y"], report=rep)
    for name in ("x", "xn1", "h1", "xn2"):
        ok &= check(name, host_f64(saved[name])[:, rows], ref[name], report=rep)
    for name in ("q", "k", "v", "ctx", "gate", "up", "act", "prod"):
        ok &= check(name, host_f64(saved[name])[:, m], ref[name], report=rep)
    ok &= check("lse", host_f64(saved["lse"])[:, :, m], ref["lse"], bf16=False, report=rep)
    assert ok, "\n".join(rep)


def test_full_size_layer_backward_last_rows():
    w = W.LLAMA2_7B
    n_last = 32
    print(f"\n[full-size backward {w.name}] dx at the last {n_last} rows", flush=True)
    buf = Buffers(w)
    buf.run(keep_stash=False)
    sh, wts, x, dy, peers = host_inputs(buf)
    ref = OL.layer_backward_last_rows(sh, wts, x, dy, n_last, peers)
    rep = []
    assert check("dx", host_f64(buf.dx)[:, -n_last:], ref, report=rep), "\n".join(rep)


def test_full_size_lm_head_at_sampled_tokens():
    w = W.LLAMA3_8B_LM_TP4
    print(f"\n[full-size LM head] N={w.tokens} h={w.hidden} v_t={w.v_t} tp={w.tp}", flush=True)
    inp = W.lm_head_inputs(w)
    loss, dh, _ = run_lm(w, inp)
    tok = sample_rows(w.tokens, k=16)
    ref = OLM.lm_head_xent(from_bits(inp["hidden"][tok]), from_bits(inp["w_lm"]), inp["targets"][tok],
                           w.tp_rank * w.v_t, inp["peer_lse"][tok], inp["peer_target_logit"][tok], 1.0 / w.tokens)
    rep, ok = [], True
    ok &= check("loss", host_f64(loss)[tok], ref["loss"], bf16=False, report=rep)
    ok &= check("d_hidden", host_f64(dh)[tok], ref["d_hidden"], report=rep)
    assert ok, "\n".join(rep)
