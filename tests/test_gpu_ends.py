"""GPU parity of the ends of the model (embedding_fwd/bwd, lm_head_fwd/bwd)
against the oracle (oracle/ends.py), and their stash bytes against Sec. 3.2.

Bar: the embedding output is bit-exact (a copy of a table row, plus a
receipt of zero, or a receipt plus zero); the table gradient is fp32 (relative
Frobenius 5e-3), and bit-exact on every row that one token alone touches;
LM-head: bf16 outputs (dx, the d(xn) sent to the peers) and fp32 outputs
(loss, softmax, gain and head-weight gradients) to the bar of gpu_common,
with the loss within 1e-3 absolute and dx given the flip allowance of the
stored d(xn) it is computed from.  The whole Llama-3-8B TP4 head is compared
in test_gpu_full_size.  The LM-head stash holds
4 s_c b h (1 + v/h) / t bytes, the LM-head term of Sec. 3.2 divided by tc;
the embedding stash holds the 8 b s_c bytes of int64 ids.
"""
import numpy as np
import pytest
import torch

import paper_2411_06465_amd as L
import workloads as W
from oracle import ends as OE
from oracle.bf16 import from_bits
from oracle.layer import Shard
from gpu_common import bf16_ulp, check, dev_bf16, host_f64

pytestmark = pytest.mark.gpu

CASES = [W.ENDS_TINY, W.ENDS_TP2CP2_RAGGED, W.ENDS_MID, W.ENDS_RAGGED_VOCAB]


def shard_of(w):
    return Shard(hidden=w.hidden, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, ffn=w.ffn, seq=w.seq,
                 micro_batch=w.micro_batch, tp=w.tp, cp=w.cp, tp_rank=w.tp_rank, cp_rank=w.cp_rank,
                 rms_eps=w.rms_eps)


def arena_for(w, extra=0):
    need = 2 * w.tokens * w.v_t * 4 + 16 * w.tokens * w.hidden + extra + (16 << 20)
    buf = torch.empty(need, dtype=torch.uint8, device="cuda")
    return L.Arena.on(buf), buf


def view(buf, stash, name, shape, dtype):
    ptr, nbytes = stash.tensor(name)
    off = ptr - buf.data_ptr()
    return buf[off:off + nbytes].view(dtype).view(shape)


def dev_opt(inp, key, fn=dev_bf16):
    return fn(inp[key]) if key in inp else None


def f32dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_embedding_matches_oracle(w):
    print(f"\n[embedding {w.name}] h={w.hidden} v_t={w.v_t} tokens={w.tokens} tp={w.tp} cp={w.cp}", flush=True)
    inp = W.ends_inputs(w)
    model, par = L.make_model(**w.model()), L.make_parallel(**w.parallel())
    arena, buf = arena_for(w)
    ids = torch.from_numpy(inp["ids"]).cuda()
    wt = dev_bf16(inp["w_emb"])
    x_out = torch.empty((w.micro_batch, w.s_sp, w.hidden), dtype=torch.bfloat16, device="cuda")
    send = torch.empty((w.micro_batch, (w.tp - 1) * w.s_sp, w.hidden), dtype=torch.bfloat16,
                       device="cuda") if w.tp > 1 else None
    rc = dev_bf16(inp["emb_receipt"]) if w.tp > 1 else None
    st = L.embedding_fwd(model, par, ids, wt, x_out, arena, receipt=rc, send=send)
    b = st.bytes()
    assert b["formula"] == 8 * w.tokens and b["aux"] == 0
    kept = view(buf, st, "ids", (w.micro_batch, w.s_c), torch.int64).cpu().numpy()
    np.testing.assert_array_equal(kept, inp["ids"])
    dw = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    L.embedding_bwd(model, par, st, dev_bf16(inp["dx_emb"]), dw, arena, peer_dx=dev_opt(inp, "peer_dx_emb"))
    torch.cuda.synchronize()
    assert arena.stats()["in_use"] == 0
    sh, v0 = shard_of(w), w.tp_rank * w.v_t
    ref = OE.embedding_forward(sh, from_bits(inp["w_emb"]), inp["ids"], v0,
                               receipt=from_bits(inp["emb_receipt"]) if w.tp > 1 else None)
    np.testing.assert_array_equal(host_f64(x_out), ref["own"])
    if w.tp > 1:
        np.testing.assert_array_equal(host_f64(send), ref["send"])
    dref = OE.embedding_backward(sh, inp["ids"], from_bits(inp["dx_emb"]),
                                 from_bits(inp["peer_dx_emb"]) if w.tp > 1 else None, w.v_t, v0)
    got = host_f64(dw)
    assert check("d_w_emb", got, dref, bf16=False)
    local = inp["ids"].reshape(-1) - v0
    local = local[(local >= 0) & (local < w.v_t)]
    u, c = np.unique(local, return_counts=True)
    once = u[c == 1]
    np.testing.assert_array_equal(got[once], dref[once])
    untouched = np.setdiff1d(np.arange(w.v_t), u)
    assert not got[untouched].any()
    arena.destroy()


def run_head(w, inp, grad_scale):
    model, par = L.make_model(**w.model()), L.make_parallel(**w.parallel())
    arena, buf = arena_for(w)
    x = dev_bf16(inp["x"])
    wn, wl = dev_bf16(inp["w_norm"]), dev_bf16(inp["w_lm"])
    tg = torch.from_numpy(inp["targets"]).cuda()
    loss = torch.empty(w.tokens, dtype=torch.float32, device="cuda")
    peer_xn = dev_opt(inp, "peer_xn")
    pl = f32dev(inp["peer_lse"]) if "peer_lse" in inp else None
    pz = f32dev(inp["peer_target_logit"]) if "peer_target_logit" in inp else None
    st = L.lm_head_fwd(model, par, x, wn, wl, tg, loss, arena, peer_xn=peer_xn, peer_lse=pl, peer_target_logit=pz)
    out = {"bytes": st.bytes()}
    out["xn"] = view(buf, st, "xn", (w.micro_batch, w.s_sp, w.hidden), torch.bfloat16).clone()
    out["probs"] = view(buf, st, "probs", (w.tokens, w.v_t), torch.float32).clone()
    out["x_kept"] = view(buf, st, "x", (w.micro_batch, w.s_sp, w.hidden), torch.bfloat16).clone()
    dx = torch.empty_like(x)
    dgn = torch.zeros(w.hidden, dtype=torch.float32, device="cuda")
    dwl = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    send = torch.empty((w.micro_batch, (w.tp - 1) * w.s_sp, w.hidden), dtype=torch.bfloat16,
                       device="cuda") if w.tp > 1 else None
    L.lm_head_bwd(model, par, wn, wl, tg, st, dx, dgn, dwl, arena, grad_scale=grad_scale, peer_xn=peer_xn,
                  peer_dxn=dev_opt(inp, "peer_dxn"), dxn_send=send)
    torch.cuda.synchronize()
    assert arena.stats()["in_use"] == 0
    arena.destroy()
    out.update(loss=loss, dx=dx, d_gain=dgn, d_w=dwl, send=send)
    return out


def head_oracle(w, inp, grad_scale):
    sh, v0 = shard_of(w), w.tp_rank * w.v_t
    x = from_bits(inp["x"])
    gain, wl = from_bits(inp["w_norm"]), from_bits(inp["w_lm"])
    tg = inp["targets"].reshape(w.micro_batch, w.s_c)
    fw = OE.lm_head_forward(sh, x, gain, wl, tg, v0, peer_xn=from_bits(inp["peer_xn"]) if w.tp > 1 else None,
                            peer_lse=inp.get("peer_lse"), peer_target_logit=inp.get("peer_target_logit"))
    bw = OE.lm_head_backward(sh, x, gain, wl, tg, v0, fw, grad_scale,
                             peer_dxn=from_bits(inp["peer_dxn"]) if w.tp > 1 else None)
    return fw, bw


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_lm_head_block_matches_oracle(w):
    print(f"\n[lm head block {w.name}] h={w.hidden} v_t={w.v_t} tokens={w.tokens} tp={w.tp} cp={w.cp}", flush=True)
    inp = W.ends_inputs(w)
    gs = 1.0 / w.tokens
    got = run_head(w, inp, gs)
    b = got["bytes"]
    # 4 s_c b h (1 + v/h) / t: x and xn (2 b s_sp h each) and the FP32 softmax (4 b s_c v_t)
    assert b["formula"] == 4 * w.s_c * w.micro_batch * (w.hidden + w.vocab) // w.tp
    assert b["aux"] == 0
    fw, bw = head_oracle(w, inp, gs)
    assert torch.equal(got["x_kept"].view(torch.int16).cpu(), torch.from_numpy(inp["x"].view(np.int16)))
    rep, ok = [], True
    ok &= check("xn", host_f64(got["xn"]), fw["xn"], contraction=False, report=rep)
    ok &= check("loss", host_f64(got["loss"]), fw["loss"], bf16=False, abs_bound=1e-3, report=rep)
    ok &= check("probs", host_f64(got["probs"]), fw["probs"], bf16=False, report=rep)
    x = from_bits(inp["x"])
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + w.rms_eps)
    # dx = RMSNorm'(d(xn)) with d(xn) stored bf16: one flip of d(xn) moves dx by |g| rstd u(d(xn))
    ok &= check("dx", host_f64(got["dx"]), bw["dx"],
                allow=np.abs(from_bits(inp["w_norm"])) * rstd * bf16_ulp(bw["d_xn"]), report=rep)
    ok &= check("d_gain", host_f64(got["d_gain"]), bw["d_gain"], bf16=False, report=rep)
    ok &= check("d_w_lm", host_f64(got["d_w"]), bw["d_w"], bf16=False, report=rep)
    if w.tp > 1:
        ok &= check("dxn_send", host_f64(got["send"]), bw["send"], report=rep)
    assert ok, "\n".join(rep)
