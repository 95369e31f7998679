"""GPU parity at the full shard sizes the benchmark runs, on whole tensors:
the Llama-2-7B layer, the Llama-3-8B TP2 CP2 and Llama-3-70B TP8 layer shards
(forward and backward: every stashed tensor, the attention LSE, y, dx, all six
weight gradients, the remote dK/dV and the four sends), and the Llama-3-8B TP4
LM head in both forms (lm_head_xent with bf16 logits; the LM-head block with
its FP32 softmax stash).  The library runs in the same launch configuration as
bench.py; the oracle runs the whole workload (float64, about 10-40 s each on
a 16-thread host).

Bar: gpu_common's, element by element (bf16 outputs within 2e-2 plus one bf16
step, plus the flip allowance of the stored operand that feeds the element
directly, plus for contraction outputs 6 x 5e-3 of the row's RMS; every tensor
within relative Frobenius 5e-3 and per-row relative error 2e-2; LSE and loss
within 2e-2 absolute); the stash byte counts equal
Eq. 12 / (tc) and the LM-head term / (tc) exactly.  With L4D_PARITY_REPORT set,
every tensor's line is appended to that file.
"""
import time

import numpy as np
import pytest
import torch

import workloads as W
from oracle import ends as OE
from oracle import lm_head as OLM
from oracle import memory as OM
from oracle.bf16 import from_bits
from gpu_common import (MAX_ABS, Buffers, bf16_ulp, check, compare_layer, host_f64, keep_report,
                        oracle_layer)
from test_gpu_ends import head_oracle, run_head
from test_gpu_lm_head import run_lm

pytestmark = pytest.mark.gpu

LAYERS = [W.LLAMA2_7B, W.LLAMA3_8B_TP2CP2, W.LLAMA3_70B_TP8]


def _say(msg, t0):
    print(f"  {msg} ({time.perf_counter() - t0:.1f} s)", flush=True)


@pytest.mark.parametrize("w", LAYERS, ids=lambda w: w.name)
def test_full_size_layer_matches_oracle(w):
    title = (f"[full-size layer {w.name}] h={w.hidden} heads={w.a_t}/{w.k_t} f_t={w.f_t} s_c={w.s_c} "
             f"tp={w.tp}/{w.tp_rank} cp={w.cp}/{w.cp_rank} b={w.micro_batch}")
    print("\n" + title, flush=True)
    t0 = time.perf_counter()
    buf = Buffers(w)
    saved = buf.run(keep_stash=True)
    _say("library forward + backward done", t0)
    assert saved["_bytes"]["formula"] == OM.act_bytes_per_layer(
        w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.seq, w.micro_batch, w.tp, w.cp)
    fw, bw = oracle_layer(w, buf.wbits, buf.abits)
    _say("oracle forward + backward done", t0)
    ok, rep = compare_layer(w, buf, saved, fw, bw)
    keep_report(title, rep)
    assert ok, "\n".join(rep)


def test_full_size_lm_head_xent_matches_oracle():
    w = W.LLAMA3_8B_LM_TP4
    title = f"[full-size lm_head_xent {w.name}] N={w.tokens} h={w.hidden} v_t={w.v_t} tp={w.tp}/{w.tp_rank}"
    print("\n" + title, flush=True)
    t0 = time.perf_counter()
    inp = W.lm_head_inputs(w)
    loss, dh, dw = run_lm(w, inp)
    _say("library done", t0)
    v0 = w.tp_rank * w.v_t
    ref = OLM.lm_head_xent(from_bits(inp["hidden"]), from_bits(inp["w_lm"]), inp["targets"], v0,
                           inp["peer_lse"], inp["peer_target_logit"], 1.0 / w.tokens)
    _say("oracle done", t0)
    # the loss subtracts the stored bf16 target logit when this shard owns the target
    local = inp["targets"] - v0
    own = (local >= 0) & (local < w.v_t)
    z = np.where(own, ref["logits"][np.arange(w.tokens), np.clip(local, 0, w.v_t - 1)], 0.0)
    rep, ok = [], True
    ok &= check("loss", host_f64(loss), ref["loss"], bf16=False, abs_bound=MAX_ABS,
                allow=np.where(own, bf16_ulp(z), 0.0), report=rep)
    ok &= check("d_hidden", host_f64(dh), ref["d_hidden"], report=rep)
    ok &= check("d_w_lm", host_f64(dw), ref["d_w"], bf16=False, report=rep)
    keep_report(title, rep)
    assert ok, "\n".join(rep)


def test_full_size_lm_head_block_matches_oracle():
    w = W.ENDS_LLAMA3_8B_TP4
    title = f"[full-size lm_head block {w.name}] tokens={w.tokens} h={w.hidden} v_t={w.v_t} tp={w.tp}/{w.tp_rank}"
    print("\n" + title, flush=True)
    t0 = time.perf_counter()
    inp = W.ends_inputs(w)
    gs = 1.0 / w.tokens
    got = run_head(w, inp, gs)
    _say("library done", t0)
    assert got["bytes"]["formula"] == 4 * w.s_c * w.micro_batch * (w.hidden + w.vocab) // w.tp
    assert torch.equal(got["x_kept"].view(torch.int16).cpu(), torch.from_numpy(inp["x"].view(np.int16)))
    fw, bw = head_oracle(w, inp, gs)
    _say("oracle done", t0)
    gain = from_bits(inp["w_norm"])
    x = from_bits(inp["x"])
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + w.rms_eps)
    rep, ok = [], True
    ok &= check("xn", host_f64(got["xn"]), fw["xn"], contraction=False, report=rep)
    ok &= check("loss", host_f64(got["loss"]), fw["loss"], bf16=False, abs_bound=MAX_ABS, report=rep)
    ok &= check("probs", host_f64(got["probs"]), fw["probs"], bf16=False, report=rep)
    # dx = RMSNorm'(d(xn)) with d(xn) stored bf16: |g| rstd u(d(xn))
    ok &= check("dx", host_f64(got["dx"]), bw["dx"], allow=np.abs(gain) * rstd * bf16_ulp(bw["d_xn"]), report=rep)
    ok &= check("d_gain", host_f64(got["d_gain"]), bw["d_gain"], bf16=False, report=rep)
    ok &= check("d_w_lm", host_f64(got["d_w"]), bw["d_w"], bf16=False, report=rep)
    if w.tp > 1:
        ok &= check("dxn_send", host_f64(got["send"]), bw["send"], report=rep)
    keep_report(title, rep)
    assert ok, "\n".join(rep)
