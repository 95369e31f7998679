"""Benchmark: one GPU's share of a Llama decoder-layer training step.

A step is one pass of the hot path on a fixed synthetic batch: the memory
estimate (host), the layer forward (which reserves the activation stash) and
the layer backward (which adds into fp32 weight-gradient accumulators).  The
headline workload is the Llama-3-70B shard at TP8 inside the (TP, CP, PP, MBS)
= (8, 1, 8, 1) layout (h 8192, 8 q / 1 kv heads per GPU, FFN shard 3584 of
28672, seq 8192, micro-batch 1).  The Llama-3-8B shard at TP2 CP2 and the
Llama-2-7B layer follow under "other_workloads" with the same per-kernel
table and roofline; the Llama-3-8B LM head at TP4 is timed alongside, and
"first_stage_1f1b" plays the first pipeline stage of the 70B (t, c, p) =
(8, 1, 8) layout under 1F1B with the real kernels (10 layers x 8
micro-batches) and compares its peak live stash with the memory model's L
layers.  "optimizer_step" times the Adam update of that layout's optimizer
shard (the 1/(d c) of a rank's parameters whose fp32 master, momentum and
variance it owns, d c = 4): 30 bytes of HBM traffic per parameter, against the
HBM peak.  "model_ends" times the LM-head block (final RMSNorm, FP32 logits
kept as the softmax, cross-entropy, forward and backward) and the embedding of
the Llama-3-8B TP4 rank, with their stash bytes against the LM-head and
embedding terms of the memory model.

Throughput is model FLOPs (forward GEMMs + causal attention over the
unmasked query/key pairs, times 3 for forward + backward) per second.  Kernel
durations come from HIP events that the library records on the launch
stream: around every launch in a few untimed steps after the warm-up (the
per-kernel table, which also names the dominant kernel), and around the
dominant kernel's launches only in the timed steps (the roofline figure).

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline] [--no-others]
    python bench.py --workload NAME [--steps K] [--warmup W]   # one layer workload alone
    python bench.py --norms-cold               # the RMSNorm kernels on cache-cold buffers
    python bench.py --calibrate-copy BYTES     # a plain device copy, for HBM counter calibration
    python bench.py --optimizer-only [--steps K] [--warmup W]   # the Adam step alone

roofline.traffic is the dominant kernel's HBM bytes per launch as measured
by rocprofv3 FETCH_SIZE + WRITE_SIZE (scaled by the counters' reading for a
plain copy of known size), read from profiles/hbm_traffic_<workload>.txt; it
is null when that file has no entry for the kernel or when the kernel's
source file has changed since the counters were taken (SHA-256 mismatch).
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E, published


# ------------------------------------------------------------------ FLOP / byte accounting

def attn_pairs(w):
    """Unmasked (query, key) pairs per head for this shard: the local query at
    global position q sees the q + 1 keys at positions 0..q."""
    if w.cp == 1:
        pos = np.arange(w.seq)
    else:
        n = w.seq // (2 * w.cp)
        pos = np.concatenate([np.arange(c * n, (c + 1) * n) for c in (w.cp_rank, 2 * w.cp - 1 - w.cp_rank)])
    return int(np.sum(pos + 1))


def gemm_shapes(w):
    tok = w.micro_batch * w.s_c
    h, nq, qc, f = w.hidden, w.a_t * w.d_h, (w.a_t + 2 * w.k_t) * w.d_h, w.f_t
    return {
        "gemm_qkv": (tok, qc, h), "gemm_o": (tok, h, nq), "gemm_gate_up": (tok, 2 * f, h), "gemm_down": (tok, h, f),
        "gemm_down_dx": (tok, f, h), "gemm_down_dw": (h, f, tok), "gemm_gate_up_dx": (tok, h, 2 * f),
        "gemm_gate_up_dw": (2 * f, h, tok), "gemm_o_dx": (tok, nq, h), "gemm_o_dw": (h, nq, tok),
        "gemm_qkv_dx": (tok, h, qc), "gemm_qkv_dw": (qc, h, tok),
    }


def layer_flops(w):
    tok = w.micro_batch * w.s_c
    h, nq, qc, f = w.hidden, w.a_t * w.d_h, (w.a_t + 2 * w.k_t) * w.d_h, w.f_t
    gemm_fwd = 2 * tok * (h * qc + nq * h + h * 2 * f + f * h)
    attn_fwd = 4 * w.d_h * attn_pairs(w) * w.a_t * w.micro_batch
    return 3 * (gemm_fwd + attn_fwd), gemm_fwd, attn_fwd


def kernel_work(w):
    """Algorithmic work per launch: ('mfma', flops) or ('hbm', bytes)."""
    out = {k: ("mfma", 2 * m * n * kk) for k, (m, n, kk) in gemm_shapes(w).items()}
    _, _, attn_fwd = layer_flops(w)
    out["attn_fwd"] = ("mfma", attn_fwd)
    out["attn_bwd_dkdv"] = ("mfma", attn_fwd)          # dK, dV: half of the 2x-forward backward
    out["attn_bwd_dq"] = ("mfma", attn_fwd)            # dQ: the other half
    rows = w.micro_batch * w.s_sp
    e, g = rows * w.hidden, 2 * w.hidden
    parts = min(rows, 256) * w.hidden * 4                  # fp32 gain-gradient partials
    out["rmsnorm1_fwd"] = ("hbm", 3 * e * 2 + g)           # read x; write xn1 and the stash copy of x
    out["rmsnorm2_fwd"] = ("hbm", 2 * e * 2 + g)           # read h1; write xn2
    out["rmsnorm2_bwd"] = ("hbm", e * (2 + 4 + 2 + 2 + 4) + g + parts)   # read h1, d(xn2) f32, dy; write dh1 bf16 + f32
    out["rmsnorm1_bwd"] = ("hbm", e * (2 + 4 + 4 + 2) + g + parts)       # read x, d(xn1) f32, dh1 f32; write dx
    return out


def lm_flops(w):
    return 3 * 2 * w.tokens * w.v_t * w.hidden


# Source file of each kernel family (for the traffic table's staleness check).
KERNEL_SOURCE = {"gemm": "gemm.hip", "attn": "attention.hip", "rmsnorm": "rowwise.hip", "reduce": "rowwise.hip",
                 "rope": "rowwise.hip", "xent": "rowwise.hip", "adam": "optim.hip"}
ADAM_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_adam_70b_shard.txt")


def traffic_file(w):
    """Counter summary of one layer workload: profiles/hbm_traffic_<name>.txt."""
    return os.path.join(ROOT, "profiles", f"hbm_traffic_{w.name.replace('-', '_')}.txt")


def source_sha(kernel):
    src = KERNEL_SOURCE.get(kernel.split("_")[0])
    if src is None:
        return None
    with open(os.path.join(ROOT, "paper_2411_06465_amd", "csrc", src), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(kernel, path):
    """HBM bytes per launch from the committed counter summary, or None when
    absent or taken on a different version of the kernel's source."""
    if not os.path.exists(path):
        return None
    sha = source_sha(kernel)
    with open(path) as f:
        for line in f:
            parts = line.split()
            if len(parts) == 5 and parts[0] == "traffic" and parts[1] == kernel:
                return int(parts[2]) if parts[4] == sha else None
    return None


def calibrate_copy(nbytes):
    """A plain device-to-device copy of nbytes, five times (for the HBM counters)."""
    import torch
    torch.cuda.set_device(0)
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {nbytes} bytes x 5", flush=True)


# ------------------------------------------------------------------ runs

def run_layer(w, steps, warmup, profile):
    """Time `steps` layer steps after `warmup` ones.  profile = P > 0 runs P
    untimed steps with events around every launch first (per-kernel table),
    then times the steps with events around the dominant kernel only."""
    import torch
    import paper_2411_06465_amd as L
    import workloads as W

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)

    wb, ab = W.layer_weights(w), W.layer_activations(w)
    weights = {k: dev(v) for k, v in wb.items()}
    x, dy = dev(ab["x"]), dev(ab["dy"])
    peers = {k: dev(v) for k, v in ab["peers"].items()}
    del wb, ab
    y, dx = torch.empty_like(x), torch.empty_like(x)
    grads = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in weights.items()}
    d_rk = d_rv = None
    if w.cp > 1:
        shape = (w.micro_batch, w.seq - w.s_c, w.k_t * w.d_h)
        d_rk = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
        d_rv = torch.empty_like(d_rk)
    model, par = L.make_model(**w.model()), L.make_parallel(**w.parallel())
    fws, bws = L.l4d_layer_workspace_bytes(model, par)
    est = L.mem_estimate(model, par)
    cap = est["act_bytes_per_layer"] + 4 * w.micro_batch * w.a_t * w.s_c + max(fws, bws) + (16 << 20)
    arena = L.Arena.on(torch.empty(cap, dtype=torch.uint8, device="cuda"))

    def step():
        L.mem_estimate(model, par)
        st = L.llama_layer_fwd(model, par, weights, x, y, arena, peers=peers)
        L.llama_layer_bwd(model, par, weights, st, dy, dx, grads, arena, peers=peers, d_remote_k=d_rk,
                          d_remote_v=d_rv)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    kernels, timed, sequence = {}, {}, []
    if profile:
        # Untimed profiled steps: an event pair around every launch gives the
        # per-kernel table and picks the kernel with the largest share.
        L.l4d_profile_only(None)
        L.l4d_profile_reset()
        L.l4d_profile_enable(True)
        for _ in range(profile):
            step()
        torch.cuda.synchronize()
        L.l4d_profile_enable(False)
        kernels = L.l4d_profile_dump()
        order = L.l4d_profile_order()
        per_step = len(order) // profile
        sequence = order[:per_step]
        work = kernel_work(w)
        dom = max((k for k in kernels if k in work), key=lambda k: kernels[k][1])
        # The timed steps carry events only around that kernel (every launch's
        # event pair would add about 6 us per launch to the step).
        L.l4d_profile_reset()
        L.l4d_profile_only(dom)
        L.l4d_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if profile:
        L.l4d_profile_enable(False)
        timed = L.l4d_profile_dump()
        L.l4d_profile_only(None)
    stash = est["act_bytes_per_layer"]
    arena.destroy()
    return (t1 - t0) / steps, kernels, timed, stash, sequence


def layer_entry(w, steps, warmup):
    """One layer workload: throughput over `steps` timed steps, the per-kernel
    table, the roofline of the kernel with the largest share and the launch
    sequence of one step."""
    prof_steps = max(3, steps // 4)
    sec, kernels, timed, stash, sequence = run_layer(w, steps, warmup, profile=prof_steps)
    flops, _, _ = layer_flops(w)
    value = flops / sec / 1e12
    work = kernel_work(w)
    dom = next(iter(timed))
    launches, total_ms = timed[dom]
    avg_s = total_ms / launches / 1e3
    kind, amount = work[dom]
    if kind == "mfma":
        roof = {"bound": "mfma", "achieved": round(amount / avg_s / 1e12, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(amount / avg_s / 1e9, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom, traffic_file(w))
    roof["kernel"] = dom
    roof["avg_ms"] = round(total_ms / launches, 4)
    kern = {}
    for k, (n, ms) in sorted(kernels.items(), key=lambda kv: -kv[1][1]):
        e = {"launches_per_step": n / prof_steps, "ms_per_step": round(ms / prof_steps, 4)}
        if k in work:
            kind_k, amt = work[k]
            per_launch_s = ms / n / 1e3
            if kind_k == "mfma":
                e["tflops"] = round(amt / per_launch_s / 1e12, 1)
            else:
                e["gbs"] = round(amt / per_launch_s / 1e9, 1)
        kern[k] = e
    return {"workload": describe(w), "tflops": round(value, 2), "ms_per_step": round(sec * 1e3, 4),
            "pct_of_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2), "model_flops_per_step": flops,
            "stash_bytes_per_layer": stash, "roofline": roof, "kernels": kern,
            "kernels_note": f"per-kernel table from {prof_steps} untimed steps with events around every launch; "
                            f"the timed steps carry events around {dom} only",
            "launch_sequence": sequence}


def norms_cold(w, steps=3):
    """The RMSNorm kernels on buffers larger than the 256 MB Infinity Cache:
    the same layer shape at a micro-batch whose norm tensors exceed it, with
    events around every launch; every kernel in between evicts the cache."""
    import torch
    _, kernels, _, _, _ = run_layer(w, 1, 1, profile=steps)
    torch.cuda.empty_cache()
    work = kernel_work(w)
    out = {"workload": f"{describe(w)}; each norm tensor {w.micro_batch * w.s_sp * w.hidden * 2 / 1e6:.0f} MB",
           "kernels": {}}
    for k in sorted(kernels):
        if k.startswith("rmsnorm") or k == "reduce_gain":
            n, ms = kernels[k]
            e = {"launches_per_step": n / steps, "us_per_launch": round(ms / n * 1e3, 1)}
            if k in work:
                e["algorithmic_bytes"] = work[k][1]
                e["gbs"] = round(work[k][1] / (ms / n / 1e3) / 1e9, 1)
                e["frac_of_hbm_peak"] = round(e["gbs"] / PEAK_HBM_GBS, 4)
            out["kernels"][k] = e
    return out


def describe(w):
    return (f"{w.name}: decoder-layer shard, forward+backward, hidden {w.hidden}, {w.a_t} q / {w.k_t} kv heads per "
            f"GPU (d_h {w.d_h}), FFN shard {w.f_t} of {w.ffn}, local tokens {w.s_c} of seq {w.seq}"
            f"{f' (+{w.seq - w.s_c} remote K/V tokens)' if w.cp > 1 else ''}, micro-batch {w.micro_batch}, "
            f"TP{w.tp} CP{w.cp}, rank ({w.tp_rank}, {w.cp_rank})")


def run_first_stage_1f1b(w):
    """Stage 0 of the (t, c, p) layout of `w` under 1F1B with p micro-batches:
    its L/p layers on the real shard kernels, every stash kept until its
    micro-batch's backward.  Peak live stash bytes against the memory model."""
    import torch
    import paper_2411_06465_amd as L
    import workloads as W
    from paper_2411_06465_amd.pipeline import run_first_stage

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)

    weights = {k: dev(v) for k, v in W.layer_weights(w).items()}
    ab = W.layer_activations(w)
    x, dy = dev(ab["x"]), dev(ab["dy"])
    peers = {k: dev(v) for k, v in ab["peers"].items()}
    del ab
    grads = {k: torch.zeros(v.shape, dtype=torch.float32, device="cuda") for k, v in weights.items()}
    model, par = L.make_model(**w.model()), L.make_parallel(**w.parallel())
    est = L.mem_estimate(model, par)
    fws, bws = L.l4d_layer_workspace_bytes(model, par)
    per = est["act_bytes_per_layer"] + 4 * w.micro_batch * w.a_t * w.s_c + (1 << 16)
    arena = L.Arena.on(torch.empty(w.n_layers * per + max(fws, bws) + (64 << 20), dtype=torch.uint8, device="cuda"))
    layers, mbs = w.n_layers // w.pp, w.pp
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = run_first_stage(model, par, weights, layers, mbs, x, dy, grads, arena, peers=peers)
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0
    in_use = arena.stats()["in_use"]
    arena.destroy()
    return {
        "workload": f"{w.name}: stage 0 of {w.pp}, {layers} layers x {mbs} micro-batches of {w.micro_batch} x "
                    f"{w.seq} tokens (t{w.tp} c{w.cp})",
        "peak_live_stashes": r["peak_live_stashes"],
        "peak_stash_bytes": r["peak_formula_bytes"],
        "model_layers_bytes": w.n_layers * r["act_bytes_per_layer"],
        "equal": r["peak_formula_bytes"] == w.n_layers * r["act_bytes_per_layer"],
        "model_first_stage_act_bytes": r["first_stage_act_bytes"],
        "model_embedding_term_bytes": r["first_stage_act_bytes"] - w.n_layers * r["act_bytes_per_layer"],
        "peak_aux_lse_bytes": r["peak_aux_bytes"],
        "peak_padding_bytes": r["peak_padding_bytes"],
        "arena_peak_bytes": r["arena_peak_bytes"],
        "in_use_after": in_use,
        "seconds": round(sec, 3),
    }


ADAM_BYTES_PER_PARAM = 30     # reads grad, master, m, v (fp32); writes master, m, v (fp32), weight (bf16)


def run_optimizer_step(w, steps, warmup):
    """The Adam step over one rank's optimizer shard (fp32 gradient, master,
    momentum, variance; bf16 weight), `steps` launches after `warmup`, with
    events around every launch on the launch stream."""
    import torch
    import paper_2411_06465_amd as L
    import workloads as W

    st = W.adam_inputs_device(w.name, w.n)
    wb = torch.empty(w.n, dtype=torch.bfloat16, device="cuda")
    hp = dict(lr=w.lr, beta1=w.beta1, beta2=w.beta2, eps=w.eps, weight_decay=w.weight_decay)
    t = w.step
    for _ in range(warmup):
        L.l4d_adam_step(st["grad"], st["master"], st["m"], st["v"], wb, t, **hp)
        t += 1
    torch.cuda.synchronize()
    L.l4d_profile_reset()
    L.l4d_profile_only("adam_step")
    L.l4d_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        L.l4d_adam_step(st["grad"], st["master"], st["m"], st["v"], wb, t, **hp)
        t += 1
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / steps
    L.l4d_profile_enable(False)
    launches, ms = L.l4d_profile_read("adam_step")
    L.l4d_profile_only(None)
    del st, wb
    torch.cuda.empty_cache()
    avg_s = ms / launches / 1e3
    gbs = ADAM_BYTES_PER_PARAM * w.n / avg_s / 1e9
    return {"workload": f"{w.name}: {w.n} parameters, Adam step {w.step}+ (lr {w.lr}, betas ({w.beta1}, "
                        f"{w.beta2}), eps {w.eps}, weight decay {w.weight_decay})",
            "bytes_per_param": ADAM_BYTES_PER_PARAM, "launches": launches,
            "kernel_ms": round(ms / launches, 4), "wall_ms_per_step": round(sec * 1e3, 4),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": measured_traffic("adam_step", ADAM_TRAFFIC_FILE)}}


def run_model_ends(w, steps, warmup):
    """The LM-head block (final RMSNorm, FP32 logits, cross-entropy; forward +
    backward) and the vocabulary-parallel embedding (forward + backward) of one
    rank, timed over `steps` after `warmup`, with their stash bytes against the
    activation terms of the memory model."""
    import torch
    import paper_2411_06465_amd as L
    import workloads as W

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)

    inp = W.ends_inputs(w)
    model, par = L.make_model(**w.model()), L.make_parallel(**w.parallel())
    buf = torch.empty(2 * w.tokens * w.v_t * 4 + 16 * w.tokens * w.hidden + (64 << 20), dtype=torch.uint8,
                      device="cuda")
    arena = L.Arena.on(buf)
    x, wn, wl = dev(inp["x"]), dev(inp["w_norm"]), dev(inp["w_lm"])
    tg = torch.from_numpy(inp["targets"]).cuda()
    peer_xn = dev(inp["peer_xn"]) if w.tp > 1 else None
    pl = torch.from_numpy(inp["peer_lse"]).cuda() if w.tp > 1 else None
    pz = torch.from_numpy(inp["peer_target_logit"]).cuda() if w.tp > 1 else None
    pdxn = dev(inp["peer_dxn"]) if w.tp > 1 else None
    loss = torch.empty(w.tokens, dtype=torch.float32, device="cuda")
    dx = torch.empty_like(x)
    dgn = torch.zeros(w.hidden, dtype=torch.float32, device="cuda")
    dwl = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    send = torch.empty((w.micro_batch, (w.tp - 1) * w.s_sp, w.hidden), dtype=torch.bfloat16,
                       device="cuda") if w.tp > 1 else None
    ids = torch.from_numpy(inp["ids"]).cuda()
    we = dev(inp["w_emb"])
    xe = torch.empty_like(x)
    rc = dev(inp["emb_receipt"]) if w.tp > 1 else None
    dxe = dev(inp["dx_emb"])
    pdxe = dev(inp["peer_dx_emb"]) if w.tp > 1 else None
    dwe = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    sizes = {}

    def head():
        st = L.lm_head_fwd(model, par, x, wn, wl, tg, loss, arena, peer_xn=peer_xn, peer_lse=pl,
                           peer_target_logit=pz)
        sizes["head"] = st.bytes()["formula"]
        L.lm_head_bwd(model, par, wn, wl, tg, st, dx, dgn, dwl, arena, grad_scale=1.0 / w.tokens,
                      peer_xn=peer_xn, peer_dxn=pdxn, dxn_send=send)

    def emb():
        st = L.embedding_fwd(model, par, ids, we, xe, arena, receipt=rc, send=send)
        sizes["emb"] = st.bytes()["formula"]
        L.embedding_bwd(model, par, st, dxe, dwe, arena, peer_dx=pdxe)

    out = {}
    for name, fn in (("lm_head_block", head), ("embedding", emb)):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        out[name] = (time.perf_counter() - t0) / steps
    arena.destroy()
    flops = 3 * 2 * w.tokens * w.v_t * w.hidden
    sbh_tc = w.seq * w.micro_batch * w.hidden // (w.tp * w.cp)
    return {"workload": f"{w.name}: {w.tokens} tokens, hidden {w.hidden}, vocabulary shard {w.v_t} of {w.vocab} "
                        f"(t{w.tp} c{w.cp})",
            "lm_head_block_ms": round(out["lm_head_block"] * 1e3, 4),
            "lm_head_block_tflops": round(flops / out["lm_head_block"] / 1e12, 1),
            "lm_head_stash_bytes": sizes["head"],
            "model_lm_head_term_bytes": 4 * sbh_tc * (w.hidden + w.vocab) // w.hidden,
            "embedding_ms": round(out["embedding"] * 1e3, 4),
            "embedding_stash_bytes": sizes["emb"],
            "model_embedding_term_bytes_per_micro_batch": 8 * sbh_tc}


def run_lm(w, steps, warmup):
    import torch
    import paper_2411_06465_amd as L
    import workloads as W

    inp = W.lm_head_inputs(w)
    hid = torch.from_numpy(inp["hidden"].view(np.int16)).cuda().view(torch.bfloat16)
    wl = torch.from_numpy(inp["w_lm"].view(np.int16)).cuda().view(torch.bfloat16)
    tg = torch.from_numpy(inp["targets"]).cuda()
    pl = torch.from_numpy(inp["peer_lse"]).cuda() if "peer_lse" in inp else None
    pz = torch.from_numpy(inp["peer_target_logit"]).cuda() if "peer_target_logit" in inp else None
    loss = torch.empty(w.tokens, dtype=torch.float32, device="cuda")
    dh = torch.empty_like(hid)
    dw = torch.zeros((w.v_t, w.hidden), dtype=torch.float32, device="cuda")
    arena = L.Arena.on(torch.empty(L.l4d_lm_head_workspace_bytes(w.tokens, w.hidden, w.v_t) + (1 << 20),
                                   dtype=torch.uint8, device="cuda"))

    def step():
        L.lm_head_xent(hid, wl, tg, loss, dh, dw, arena, vocab_start=w.tp_rank * w.v_t, peer_lse=pl,
                       peer_target_logit=pz, grad_scale=1.0 / w.tokens)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, seq):
    """The oracle (float64 numpy, as written) on a bounded sample of the same
    shard: the same hidden size, heads, FFN shard and (TP, CP) layout at global
    sequence `seq` instead of the workload's (the default keeps it to 10-30 s
    of CPU work)."""
    from threadpoolctl import threadpool_info
    import workloads as W
    from oracle import layer as OL
    from oracle.bf16 import from_bits

    ws = w.replace(name=w.name + "-cpu-sample", seq=seq)
    wb, ab = W.layer_weights(ws), W.layer_activations(ws)
    sh = OL.Shard(**ws.shard_kwargs())
    wts = {k: from_bits(v) for k, v in wb.items()}
    x, dy = from_bits(ab["x"]), from_bits(ab["dy"])
    peers = {k: from_bits(v) for k, v in ab["peers"].items()}
    t0 = time.perf_counter()
    fw = OL.layer_forward(sh, wts, x, peers)
    OL.layer_backward(sh, wts, fw, dy, peers)
    dt = time.perf_counter() - t0
    flops, _, _ = layer_flops(ws)
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(flops / dt / 1e12, 5), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "logical_cpus": os.cpu_count(),
            "sample": f"{ws.name}: one shard fwd+bwd at global seq {seq}"
                      f"{' (the whole workload)' if seq == w.seq else f' of the workload {w.seq}'} (h {w.hidden}, "
                      f"{w.a_t}/{w.k_t} heads and FFN shard {w.f_t} per rank, TP{w.tp} CP{w.cp}), "
                      f"{flops / 1e12:.3f} TFLOP, float64 numpy, {dt:.1f} s wall"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-others", action="store_true")
    ap.add_argument("--cpu-seq", type=int, default=8192,
                    help="sequence of the oracle's CPU sample of the headline shard (8192: the whole workload)")
    ap.add_argument("--workload", default="", help="time one layer workload alone and print its object")
    ap.add_argument("--norms-cold", action="store_true",
                    help="time only the RMSNorm kernels on cache-cold buffers and print that object")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES")
    ap.add_argument("--optimizer-only", action="store_true",
                    help="time only the Adam step over the 70B optimizer shard and print its object")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU's shard: the library has no multi-GPU path; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as W
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.optimizer_only:
        print(json.dumps({"optimizer_step": run_optimizer_step(W.ADAM_70B_SHARD, args.steps, args.warmup)}),
              flush=True)
        return

    cold = W.LLAMA2_7B.replace(name="llama2-7b-layer-b8", micro_batch=8)
    if args.norms_cold:
        print(json.dumps({"memory_bound_cold": norms_cold(cold)}), flush=True)
        return
    layers = {lw.name: lw for lw in (W.LLAMA3_70B_TP8, W.LLAMA3_8B_TP2CP2, W.LLAMA2_7B)}
    if args.workload:
        if args.workload not in layers:
            print(f"unknown workload {args.workload}; one of {sorted(layers)}", file=sys.stderr)
            sys.exit(2)
        print(json.dumps({args.workload: layer_entry(layers[args.workload], args.steps, args.warmup)}), flush=True)
        return

    # Headline: the Llama-3-70B shard at TP8 (the largest layer shard, and a
    # target shape); the Llama-3-8B TP2 CP2 shard and the Llama-2-7B layer
    # follow with the same per-kernel table and roofline.
    w = W.LLAMA3_70B_TP8
    head = layer_entry(w, args.steps, args.warmup)
    torch.cuda.empty_cache()
    out = {
        "metric": "TFLOP/s per GPU, Llama layer fwd+bwd shard; % of bf16 MFMA peak",
        "value": head["tflops"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": head["workload"], "global_batch": w.micro_batch, "seq_len": w.seq,
                   "parallelism": f"tp{w.tp}-cp{w.cp}-pp{w.pp} shard (one rank of {w.n_gpus})",
                   "model_flops_per_step": head["model_flops_per_step"],
                   "stash_bytes_per_layer": head["stash_bytes_per_layer"]},
        "pct_of_bf16_peak": head["pct_of_bf16_peak"],
        "roofline": head["roofline"],
        "kernels": head["kernels"],
        "kernels_note": head["kernels_note"],
        "launch_sequence": head["launch_sequence"],
    }

    if not args.no_others:
        others = {}
        for ow in (W.LLAMA3_8B_TP2CP2, W.LLAMA2_7B):
            others[ow.name] = layer_entry(ow, args.steps, args.warmup)
            torch.cuda.empty_cache()
        lw = W.LLAMA3_8B_LM_TP4
        s3 = run_lm(lw, max(5, args.steps // 2), 2)
        others[lw.name] = {"tflops": round(lm_flops(lw) / s3 / 1e12, 2), "ms_per_step": round(s3 * 1e3, 3),
                           "pct_of_bf16_peak": round(100 * lm_flops(lw) / s3 / 1e12 / PEAK_BF16_TFLOPS, 2)}
        out["other_workloads"] = others
        # the memory-bound kernels on cold buffers (the Llama-2-7B layer at micro-batch 8)
        out["memory_bound_cold"] = norms_cold(cold)
        torch.cuda.empty_cache()
        # the paper's first-stage claim, measured: 80 layer stashes of the 70B TP8 shard
        out["first_stage_1f1b"] = run_first_stage_1f1b(W.LLAMA3_70B_TP8)
        torch.cuda.empty_cache()
        # the ends of the model: LM-head block with its FP32 softmax stash, and the embedding
        out["model_ends"] = run_model_ends(W.ENDS_LLAMA3_8B_TP4, max(5, args.steps // 2), 2)
        torch.cuda.empty_cache()
        # the per-step optimizer update of the same layout's optimizer shard
        out["optimizer_step"] = run_optimizer_step(W.ADAM_70B_SHARD, max(10, args.steps // 2), 3)

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seq)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
