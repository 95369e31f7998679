"""GPU parity of the layer shard (forward + backward) against the oracle.

Every case runs the HIP library through its C ABI on seeded inputs and the
CPU oracle on the same bytes, then compares every stashed tensor, every output
and every weight gradient to the parity bar of gpu_common (bf16 tensors: every
element within 2e-2 plus one bf16 step, plus the flip allowance of the stored
operand that feeds it directly, plus for contraction outputs 6 x 5e-3 of the
row's RMS; every tensor: relative Frobenius <= 5e-3 and per-row relative error
<= 2e-2; the attention LSE within 2e-2 absolute).
The stash byte count must equal Eq. 12 / (tc) exactly.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import memory as OM
from gpu_common import Buffers, compare_layer, oracle_layer

pytestmark = pytest.mark.gpu

T = W.TINY
CASES = {
    "tiny": T,
    "tiny-b2": T.replace(name="tiny-b2", micro_batch=2),
    "tiny-tp2-r1": T.replace(name="tiny-tp2", tp=2, tp_rank=1, n_gpus=2),
    "tiny-cp2-r1": T.replace(name="tiny-cp2", cp=2, cp_rank=1, n_gpus=2),
    "tiny-tp2cp2": T.replace(name="tiny-tp2cp2", tp=2, cp=2, tp_rank=1, cp_rank=0, n_gpus=4, micro_batch=2),
    "ragged-s200": T.replace(name="ragged-s200", seq=200),
    "d128-s384": W.LayerWorkload("d128-s384", 512, 4, 2, 1376, 384, rope_base=5e5),
    "gqa8-cp2-s320": W.LayerWorkload("gqa8-cp2", 1024, 8, 1, 512, 320, cp=2, cp_rank=0, n_gpus=2, rope_base=5e5),
    "mha-cp4-r2": W.LayerWorkload("mha-cp4", 512, 4, 4, 768, 512, cp=4, cp_rank=2, n_gpus=4, rope_base=1e4),
    # 1024 tokens over few weight-gradient tiles: those GEMMs cut their token range in 4 parts
    # (d128-s384: in 3), each part summed in fp32 and added to the accumulator in order
    "d128-s1024-splitk": W.LayerWorkload("d128-s1024", 512, 4, 2, 1376, 1024, rope_base=5e5),
    # GQA group 4 per rank at TP2 (dK/dV split over query heads) with split weight gradients
    "gqa4-tp2-s768": W.LayerWorkload("gqa4-tp2", 1024, 8, 2, 2816, 768, tp=2, tp_rank=0, n_gpus=2, rope_base=5e5),
    # CP2 with two sequences per micro-batch: remote key segments in the heaviest-first dK/dV order
    "cp2-b2-s1024": W.LayerWorkload("cp2-b2", 512, 4, 4, 1376, 1024, micro_batch=2, cp=2, cp_rank=1, n_gpus=2,
                                    rope_base=1e4),
}


@pytest.mark.parametrize("name", list(CASES))
def test_layer_matches_oracle(name):
    w = CASES[name]
    print(f"\n[case {name}] h={w.hidden} a={w.n_heads} k={w.n_kv_heads} f={w.ffn} s={w.seq} "
          f"b={w.micro_batch} tp={w.tp}/{w.tp_rank} cp={w.cp}/{w.cp_rank}", flush=True)
    buf = Buffers(w)
    saved = buf.run()
    fw, bw = oracle_layer(w, buf.wbits, buf.abits)

    assert saved["_bytes"]["formula"] == OM.act_bytes_per_layer(
        w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.seq, w.micro_batch, w.tp, w.cp)

    ok, rep = compare_layer(w, buf, saved, fw, bw)
    assert ok, "\n".join(rep)


@pytest.mark.parametrize("name", ["tiny-cp2-r1", "d128-s384"])
def test_layer_is_deterministic_and_accumulates_gradients(name):
    w = CASES[name]
    buf = Buffers(w)
    buf.run(keep_stash=False)
    y1, dx1 = buf.y.clone(), buf.dx.clone()
    g1 = {k: v.clone() for k, v in buf.grads.items()}
    buf.run(keep_stash=False)
    assert torch.equal(buf.y, y1) and torch.equal(buf.dx, dx1)
    for k in g1:     # the backward adds into the accumulators
        assert torch.allclose(buf.grads[k], 2 * g1[k], rtol=1e-6, atol=1e-6), k
    assert buf.arena.stats()["in_use"] == 0


def test_zero_output_projections_give_identity_on_gpu():
    # W_O = W_down = 0: y == x and dx == dy bit for bit (a special case of the layer)
    w = CASES["tiny-b2"]
    buf = Buffers(w)
    buf.weights["o"].zero_()
    buf.weights["down"].zero_()
    buf.run(keep_stash=False)
    assert torch.equal(buf.y, buf.x)
    assert torch.equal(buf.dx, buf.dy)
