"""GPU parity of the TP-sharded LM head + vocabulary-parallel cross-entropy."""
import numpy as np
import pytest
import torch

import paper_2411_06465_amd as L
import workloads as W
from oracle import lm_head as OLM
from oracle.bf16 import from_bits
from gpu_common import check, dev_bf16, host_f64

pytestmark = pytest.mark.gpu

CASES = {
    "t1-small": W.LMHeadWorkload("lm-t1", 256, 256, 1000),
    "t4-ragged": W.LMHeadWorkload("lm-t4", 300, 512, 4000, tp=4, tp_rank=2),
    # vocabulary shard 1288: d_hidden over the first 1280 on the BK = 64 kernel, the last 8 on the ragged one
    "t2-split-k": W.LMHeadWorkload("lm-t2", 512, 512, 2576, tp=2, tp_rank=1),
}


def run_lm(w, inp, w_lm=None):
    hid = dev_bf16(inp["hidden"])
    wl = dev_bf16(inp["w_lm"]) if w_lm is None else w_lm
    tg = torch.from_numpy(inp["targets"]).cuda()
    pl = torch.from_numpy(inp["peer_lse"]).cuda() if "peer_lse" in inp else None
    pz = torch.from_numpy(inp["peer_target_logit"]).cuda() if "peer_target_logit" in inp else None
    loss = torch.empty(w.tokens, dtype=torch.float32, device="cuda")
    dh = torch.empty_like(hid)
    dw = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    buf = torch.empty(L.l4d_lm_head_workspace_bytes(w.tokens, w.hidden, w.v_t) + (1 << 20), dtype=torch.uint8,
                      device="cuda")
    arena = L.Arena.on(buf)
    L.lm_head_xent(hid, wl, tg, loss, dh, dw, arena, vocab_start=w.tp_rank * w.v_t, peer_lse=pl,
                   peer_target_logit=pz, grad_scale=1.0 / w.tokens)
    torch.cuda.synchronize()
    assert arena.stats()["in_use"] == 0
    return loss, dh, dw


@pytest.mark.parametrize("name", list(CASES))
def test_lm_head_matches_oracle(name):
    w = CASES[name]
    print(f"\n[case {name}] N={w.tokens} h={w.hidden} v_t={w.v_t} tp={w.tp}", flush=True)
    inp = W.lm_head_inputs(w)
    loss, dh, dw = run_lm(w, inp)
    ref = OLM.lm_head_xent(from_bits(inp["hidden"]), from_bits(inp["w_lm"]), inp["targets"], w.tp_rank * w.v_t,
                           inp.get("peer_lse"), inp.get("peer_target_logit"), 1.0 / w.tokens)
    rep, ok = [], True
    ok &= check("loss", host_f64(loss), ref["loss"], bf16=False, report=rep)
    ok &= check("d_hidden", host_f64(dh), ref["d_hidden"], report=rep)
    ok &= check("d_w_lm", host_f64(dw), ref["d_w"], bf16=False, report=rep)
    assert ok, "\n".join(rep)


def test_lm_head_zero_weight_gives_ln_v():
    # W_lm = 0 and peer LSE = ln(v - v_t): every loss is ln v (the closed form of the oracle pin)
    w = W.LMHeadWorkload("lm-zero", 64, 256, 4096, tp=4, tp_rank=1)
    inp = W.lm_head_inputs(w)
    inp["peer_lse"] = np.full(w.tokens, np.log(w.vocab - w.v_t), dtype=np.float32)
    inp["peer_target_logit"] = np.zeros(w.tokens, dtype=np.float32)
    zero = torch.zeros((w.v_t, w.hidden), dtype=torch.bfloat16, device="cuda")
    loss, dh, dw = run_lm(w, inp, w_lm=zero)
    assert np.allclose(loss.cpu().numpy(), np.log(w.vocab), rtol=1e-6)
    assert torch.count_nonzero(dh) == 0
