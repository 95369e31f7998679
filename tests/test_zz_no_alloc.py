"""lm_head_xent_noalloc (the LM head over the library's static per-GPU
workspace) against lm_head_xent (the same kernels over an arena): two calls in
a row on one device, the second smaller than the first, so the static array
still holds the first call's logits when the second starts.  The kernels are
deterministic and the workspace is fully written before it is read, so the
outputs must be bit-identical.  A problem larger than the 64 MiB array is
rejected with L4D_EINVAL before anything is launched."""
import numpy as np
import pytest
import torch

import paper_2411_06465_amd as L
import workloads as W
from gpu_common import dev_bf16

pytestmark = pytest.mark.gpu

CALLS = [
    # vocabulary shard 1288: logits plus the fp32 sum of d_hidden (ragged tail)
    W.LMHeadWorkload("lm-noalloc-1", 512, 512, 2576, tp=2, tp_rank=1),
    # smaller: 300 tokens of a 1000-wide shard, logits only
    W.LMHeadWorkload("lm-noalloc-2", 300, 256, 4000, tp=4, tp_rank=2),
]


def _inputs(w):
    inp = W.lm_head_inputs(w)
    d = dict(hid=dev_bf16(inp["hidden"]), wl=dev_bf16(inp["w_lm"]), tg=torch.from_numpy(inp["targets"]).cuda(),
             pl=torch.from_numpy(inp["peer_lse"]).cuda() if "peer_lse" in inp else None,
             pz=torch.from_numpy(inp["peer_target_logit"]).cuda() if "peer_target_logit" in inp else None)
    return d


def _outputs(w):
    loss = torch.empty(w.tokens, dtype=torch.float32, device="cuda")
    dh = torch.empty((w.tokens, w.hidden), dtype=torch.bfloat16, device="cuda")
    dw = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    return loss, dh, dw


def test_noalloc_matches_arena_entry_point_on_two_calls():
    for w in CALLS:
        print(f"\n[no-alloc LM head {w.name}] N={w.tokens} h={w.hidden} v_t={w.v_t}", flush=True)
        d = _inputs(w)
        kw = dict(vocab_start=w.tp_rank * w.v_t, peer_lse=d["pl"], peer_target_logit=d["pz"],
                  grad_scale=1.0 / w.tokens)
        loss_a, dh_a, dw_a = _outputs(w)
        buf = torch.empty(L.l4d_lm_head_workspace_bytes(w.tokens, w.hidden, w.v_t) + (1 << 20), dtype=torch.uint8,
                          device="cuda")
        arena = L.Arena.on(buf)
        L.lm_head_xent(d["hid"], d["wl"], d["tg"], loss_a, dh_a, dw_a, arena, **kw)
        loss_n, dh_n, dw_n = _outputs(w)
        L.lm_head_xent_noalloc(d["hid"], d["wl"], d["tg"], loss_n, dh_n, dw_n, **kw)
        torch.cuda.synchronize()
        assert torch.equal(loss_n, loss_a)
        assert torch.equal(dh_n.view(torch.int16), dh_a.view(torch.int16))
        assert torch.equal(dw_n, dw_a)
        assert bool(torch.isfinite(loss_n).all()) and bool(dw_n.abs().sum() > 0)
        arena.destroy()


def test_noalloc_rejects_a_problem_larger_than_its_array():
    w = W.LMHeadWorkload("lm-noalloc-big", 2048, 4096, 128256, tp=4)     # 131 MB of logits
    hid = torch.zeros((w.tokens, w.hidden), dtype=torch.bfloat16, device="cuda")
    wl = torch.zeros((w.v_t, w.hidden), dtype=torch.bfloat16, device="cuda")
    tg = torch.zeros(w.tokens, dtype=torch.int64, device="cuda")
    pl = torch.zeros(w.tokens, dtype=torch.float32, device="cuda")
    loss, dh, dw = _outputs(w)
    with pytest.raises(L.L4DError) as e:
        L.lm_head_xent_noalloc(hid, wl, tg, loss, dh, dw, peer_lse=pl, peer_target_logit=pl)
    assert e.value.code == L.L4D_EINVAL
