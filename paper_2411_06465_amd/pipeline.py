"""The first pipeline stage under 1F1B, on one GPU (Sec. 3.2.2, Eq. 16-17).

Under the one-forward-one-backward schedule a pipeline stage keeps the
activations of every micro-batch it has run forward but not yet backward.
Stage 0 runs p - 1 warm-up forwards before its first backward, so at its peak
it holds p micro-batches of its L/p layers: the activations of L layers, which
is why the memory model counts the first stage with L layers.  `run_first_stage`
plays that stage's schedule with the real layer kernels (every layer of a
micro-batch keeps its stash until that micro-batch's backward) and reports the
peak of the live stashes next to the memory model.
"""
import torch

from . import (llama_layer_bwd, llama_layer_fwd, mem_estimate)


def one_f_one_b(stage, stages, micro_batches):
    """Operation order of pipeline stage `stage` (0-based) of `stages` under 1F1B
    with a flush: stages - stage - 1 warm-up forwards, then forward / backward
    pairs, then the remaining backwards.  Returns [("F", i) | ("B", i)]."""
    if not 0 <= stage < stages or micro_batches < 1:
        raise ValueError("need 0 <= stage < stages and micro_batches >= 1")
    warm = min(stages - stage - 1, micro_batches)
    ops = [("F", i) for i in range(warm)]
    f, b = warm, 0
    while f < micro_batches:
        ops += [("F", f), ("B", b)]
        f, b = f + 1, b + 1
    ops += [("B", i) for i in range(b, micro_batches)]
    return ops


def run_first_stage(model, par, weights, layers, micro_batches, x, dy, grads, arena, peers=None,
                    d_remote_k=None, d_remote_v=None):
    """Stage 0 of par.pp stages over `micro_batches` micro-batches: a forward
    runs `layers` layers, each keeping its stash, a backward runs them in reverse
    and returns their stashes.  All layers share `weights` (a stash's size does
    not depend on the values), and every micro-batch starts from `x` and `dy`.

    Returns the peak over the schedule of the live stashes (count and bytes:
    the model's formula bytes, the LSE aux bytes, alignment padding), the
    arena's peak (stashes plus transient workspace), the memory model's
    per-layer and first-stage activation bytes, and the schedule."""
    ping, pong = torch.empty_like(x), torch.empty_like(x)
    gx, gy = torch.empty_like(dy), torch.empty_like(dy)
    live = {}                      # micro-batch -> its stashes, layer order
    peak = dict(stashes=0, formula=0, aux=0, padding=0)
    ops = one_f_one_b(0, par.pp, micro_batches)
    for op, mb in ops:
        if op == "F":
            inp, out, stashes = x, ping, []
            for _ in range(layers):
                stashes.append(llama_layer_fwd(model, par, weights, inp, out, arena, peers=peers))
                inp, out = out, (pong if out is ping else ping)
            live[mb] = stashes
            tot = dict(stashes=0, formula=0, aux=0, padding=0)
            for sts in live.values():
                for st in sts:
                    b = st.bytes()
                    tot["stashes"] += 1
                    for k in ("formula", "aux", "padding"):
                        tot[k] += b[k]
            if tot["formula"] > peak["formula"]:
                peak = tot
        else:
            grad, out = dy, gx
            for st in reversed(live.pop(mb)):
                llama_layer_bwd(model, par, weights, st, grad, out, grads, arena, peers=peers,
                                d_remote_k=d_remote_k, d_remote_v=d_remote_v)
                grad, out = out, (gy if out is gx else gx)
    est = mem_estimate(model, par)
    return dict(peak_live_stashes=peak["stashes"], peak_formula_bytes=peak["formula"],
                peak_aux_bytes=peak["aux"], peak_padding_bytes=peak["padding"],
                arena_peak_bytes=arena.stats()["peak"], act_bytes_per_layer=est["act_bytes_per_layer"],
                first_stage_act_bytes=est["act_bytes"], ops=ops)
