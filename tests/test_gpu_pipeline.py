"""The first pipeline stage under 1F1B with the real layer kernels (Sec. 3.2.2):
at its peak it holds p micro-batches of its L/p layers, i.e. exactly L times
the per-layer activation bytes of Eq. 12, and every stash goes back to the arena."""
import pytest
import torch

import paper_2411_06465_amd as L
import workloads as W
from oracle import memory as OM
from paper_2411_06465_amd.pipeline import run_first_stage

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("pp,m", [(2, 3), (4, 4)])
def test_first_stage_peak_is_L_layers(pp, m):
    w = W.TINY.replace(name="tiny-pp", pp=pp, n_gpus=pp, n_layers=4 * pp)
    print(f"\n[case tiny pp={pp} micro-batches={m} layers={w.n_layers}]", flush=True)

    def dev(bits):
        return torch.from_numpy(bits.view("int16").copy()).cuda().view(torch.bfloat16)

    weights = {k: dev(v) for k, v in W.layer_weights(w).items()}
    acts = W.layer_activations(w)
    x, dy = dev(acts["x"]), dev(acts["dy"])
    grads = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in weights.items()}
    model, par = L.make_model(**w.model()), L.make_parallel(**w.parallel())
    est = L.mem_estimate(model, par)
    fws, bws = L.l4d_layer_workspace_bytes(model, par)
    per = est["act_bytes_per_layer"] + 4 * w.micro_batch * w.a_t * w.s_c + (1 << 16)
    arena = L.Arena.on(torch.empty(w.n_layers * per + max(fws, bws) + (1 << 20), dtype=torch.uint8, device="cuda"))
    r = run_first_stage(model, par, weights, w.n_layers // pp, m, x, dy, grads, arena)
    torch.cuda.synchronize()
    # the memory model's per-layer term (Eq. 12 / (tc)), from the oracle
    layer_bytes = OM.act_bytes_per_layer(w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.seq, w.micro_batch, w.tp, w.cp)
    assert r["peak_live_stashes"] == min(pp, m) * (w.n_layers // pp)
    assert r["peak_formula_bytes"] == r["peak_live_stashes"] * layer_bytes
    if m >= pp:       # the first stage holds L layers (Eq. 16-17)
        assert r["peak_formula_bytes"] == w.n_layers * layer_bytes
    assert r["peak_aux_bytes"] == r["peak_live_stashes"] * 4 * w.micro_batch * w.a_t * w.s_c
    assert arena.stats()["in_use"] == 0
    assert all(torch.isfinite(g).all() for g in grads.values())
    arena.destroy()
