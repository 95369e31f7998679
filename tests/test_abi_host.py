"""Host-side checks of the C ABI (no GPU needed).

The library is loaded and driven through ctypes, but only its host logic runs:
symbol exports, the memory estimate, the arena / stash bookkeeping and the
argument validation.  Nothing here launches a kernel; arenas are created over
a fake device address that the host code never dereferences.
"""
import ctypes as C
import json
import os
import re

import pytest

import paper_2411_06465_amd as L
from oracle import memory as M
from workloads import LAYER_WORKLOADS, TINY, LLAMA2_7B, LLAMA3_8B_TP2CP2, LLAMA3_70B_TP8

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "l4d.h")
FAKE_BASE = 1 << 40            # never dereferenced by the host code

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="libl4d.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\**(\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert "llama_layer_fwd" in names and "mem_estimate" in names and "lm_head_xent" in names
    lib = C.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def model_par(w, **over):
    d = dict(w.model())
    d.update(over)
    p = dict(w.parallel())
    p.update({k: v for k, v in over.items() if k in p})
    return L.make_model(**d), L.make_parallel(**p)


# ------------------------------------------------------------------ memory estimate

ARCH = {"llama-3.1-8b": (4096, 32, 8, 14336, 32, 128256), "llama-3.1-70b": (8192, 64, 8, 28672, 80, 128256)}


def test_mem_estimate_equals_oracle_on_every_paper_cell():
    cells = json.load(open(os.path.join(ROOT, "tests", "golden", "paper_memory_tables.json")))["cells"]
    for c in cells:
        h, a, k, f, Lyr, v = ARCH[c["model"]]
        d = c["n_gpus"] // (c["tp"] * c["cp"] * c["pp"])
        got = L.mem_estimate(L.make_model(h, a, k, f, Lyr, v),
                             L.make_parallel(c["seq"], c["mbs"], c["tp"], c["cp"], c["pp"], d))
        want = M.estimate(h, a, k, f, Lyr, v, s=c["seq"], b=c["mbs"], t=c["tp"], c=c["cp"], p=c["pp"], d=d)
        assert got["params_per_gpu"] == want["params"]
        assert got["weight_bytes"] == want["weight"]
        assert got["grad_bytes"] == want["grad"]
        assert got["optim_bytes"] == want["optim"]
        assert got["act_bytes_per_layer"] == want["act_layer"]
        assert got["act_bytes"] == want["act"]
        assert got["total_bytes"] == want["total"]
        assert got["inexact"] == 0


@pytest.mark.parametrize("w", list(LAYER_WORKLOADS.values()), ids=lambda w: w.name)
def test_mem_estimate_equals_oracle_on_workloads(w):
    got = L.mem_estimate(*model_par(w))
    want = M.estimate(w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.n_layers, w.vocab, s=w.seq,
                      b=w.micro_batch, t=w.tp, c=w.cp, p=w.pp, d=w.dp)
    assert got["total_bytes"] == want["total"] and got["act_bytes_per_layer"] == want["act_layer"]


def test_mem_estimate_pins():
    # Appendix A.1, 70B (8,1,8,1) on 256 GPUs: 35.88 GiB; Sec. 4.2.1: 89.95 GiB
    g = L.mem_estimate(*model_par(LLAMA3_70B_TP8))
    assert g["total_bytes"] == 38_525_370_368
    g = L.mem_estimate(L.make_model(4096, 32, 8, 14336, 32, 128256), L.make_parallel(8192, 1, 1, 2, 1, 2))
    assert round(g["total_bytes"] / 2 ** 30, 2) == 89.95


def test_mem_estimate_flags_fractional_terms():
    # d*c = 3 does not divide 12 Psi for this tiny model: rounded up and flagged
    g = L.mem_estimate(L.make_model(8, 1, 1, 8, 1, 8), L.make_parallel(8, 1, 1, 1, 1, 7))
    psi = M.params_per_gpu(8, 1, 1, 8, 1, 8, 1, 1)
    assert g["params_per_gpu"] == psi
    assert g["inexact"] == (0 if (12 * psi) % 7 == 0 else 1)


@pytest.mark.parametrize("bad", [dict(n_heads=3), dict(n_kv_heads=3), dict(tp=3), dict(cp=3), dict(pp=3),
                                 dict(tp_rank=2), dict(cp_rank=-1), dict(ffn=31), dict(seq=0)])
def test_mem_estimate_rejects_bad_layouts(bad):
    base = dict(hidden=64, n_heads=4, n_kv_heads=2, ffn=32, n_layers=4, vocab=16, seq=16, tp=2, cp=2, pp=2)
    base.update(bad)
    m = L.make_model(**base)
    p = L.make_parallel(**base)
    with pytest.raises(L.L4DError) as e:
        L.mem_estimate(m, p)
    assert e.value.code == L.L4D_EINVAL


# ------------------------------------------------------------------ stash accounting

@pytest.mark.parametrize("w", list(LAYER_WORKLOADS.values()), ids=lambda w: w.name)
def test_stash_bytes_equal_the_activation_formula(w):
    m, p = model_par(w)
    want = M.act_bytes_per_layer(w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.seq, w.micro_batch, w.tp, w.cp)
    a = L.Arena(FAKE_BASE, 1 << 40)
    st = L.l4d_stash_reserve(a, m, p)
    b = st.bytes()
    assert b["formula"] == want == L.mem_estimate(m, p)["act_bytes_per_layer"]
    assert b["aux"] == 4 * w.micro_batch * w.a_t * w.s_c      # FlashAttention LSE, counted as zero
    # every tensor inside the arena block, disjoint
    spans = sorted(st.tensor(i) for i in range(len(L.STASH_NAMES)))
    for (p0, n0), (p1, _) in zip(spans, spans[1:]):
        assert p0 + n0 <= p1
    assert spans[0][0] >= FAKE_BASE
    for bad in (-1, len(L.STASH_NAMES)):     # one past the last tensor is refused, not read
        with pytest.raises(L.L4DError) as e:
            st.tensor(bad)
        assert e.value.code == L.L4D_EINVAL
    st.release()
    assert a.stats()["in_use"] == 0
    a.destroy()


def test_stash_reserve_fails_with_enomem_exactly_at_capacity():
    m, p = model_par(TINY)
    probe = L.Arena(FAKE_BASE, 1 << 30)
    st = L.l4d_stash_reserve(probe, m, p)
    need = probe.stats()["in_use"]
    st.release()
    probe.destroy()
    ok = L.Arena(FAKE_BASE, need)
    L.l4d_stash_reserve(ok, m, p).release()
    small = L.Arena(FAKE_BASE, need - 256)
    with pytest.raises(L.L4DError) as e:
        L.l4d_stash_reserve(small, m, p)
    assert e.value.code == L.L4D_ENOMEM
    assert small.stats()["in_use"] == 0


@pytest.mark.parametrize("order", ["fifo", "lifo"])
def test_arena_release_orders_restore_a_single_free_block(order):
    # 1F1B keeps up to p micro-batches of stashes alive; release in either order.
    m, p = model_par(TINY)
    a = L.Arena(FAKE_BASE, 64 << 20)
    stashes = [L.l4d_stash_reserve(a, m, p) for _ in range(8)]
    peak = a.stats()["in_use"]
    assert peak == 8 * (peak // 8)
    for st in (stashes if order == "fifo" else stashes[::-1]):
        st.release()
    assert a.stats()["in_use"] == 0 and a.stats()["peak"] == peak
    # coalesced: the whole capacity fits again
    big = L.Arena(FAKE_BASE, 64 << 20)
    sts = [L.l4d_stash_reserve(big, m, p) for _ in range(8)]
    for st in sts:
        st.release()
    a.destroy()
    big.destroy()


def test_arena_destroy_refuses_live_stash():
    m, p = model_par(TINY)
    a = L.Arena(FAKE_BASE, 64 << 20)
    st = L.l4d_stash_reserve(a, m, p)
    with pytest.raises(L.L4DError):
        a.destroy()
    st.release()
    a.destroy()


def test_workspace_sizes_are_reported():
    for w in LAYER_WORKLOADS.values():
        f, b = L.l4d_layer_workspace_bytes(*model_par(w))
        assert f > 0 and b > 0
    # bf16 logits, plus an fp32 d_hidden when the vocabulary shard is not a multiple of 128
    assert L.l4d_lm_head_workspace_bytes(8192, 4096, 32064) == 8192 * 32064 * 2 + 8192 * 4096 * 4
    assert L.l4d_lm_head_workspace_bytes(8192, 4096, 32000) == 8192 * 32000 * 2


def test_layer_calls_validate_before_touching_the_device():
    m, p = model_par(LLAMA3_8B_TP2CP2)
    a = L.Arena(FAKE_BASE, 1 << 40)
    # missing weights -> EINVAL, nothing reserved
    rc = L.lib().llama_layer_fwd(C.byref(m), C.byref(p), None, None, None, None, None, a.h, C.byref(C.c_void_p()), None)
    assert rc == L.L4D_EINVAL and a.stats()["in_use"] == 0
    # head dim 96 unsupported
    m2 = L.make_model(hidden=96 * 4, n_heads=4, n_kv_heads=4, ffn=64)
    with pytest.raises(L.L4DError):
        L.l4d_layer_workspace_bytes(m2, L.make_parallel(64))
    a.destroy()


def _adam(**kw):
    base = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0, grad_scale=1.0,
                grad_scale_dev=None, step=1, zero_grad=0)
    base.update(kw)
    return L.Adam(*[base[n] for n, _ in L.Adam._fields_])


def _adam_rc(hp, n=1024, ptrs=None):
    g, w, m, v, b = ptrs or (FAKE_BASE, FAKE_BASE + (1 << 20), FAKE_BASE + (2 << 20), FAKE_BASE + (3 << 20),
                             FAKE_BASE + (4 << 20))
    return L.lib().l4d_adam_step(C.byref(hp), n, g, w, m, v, b, None)


def test_adam_step_validates_before_touching_the_device():
    # every rejected call returns before any HIP call, so fake addresses are safe
    assert _adam_rc(_adam(step=0)) == L.L4D_EINVAL
    assert _adam_rc(_adam(beta1=1.0)) == L.L4D_EINVAL
    assert _adam_rc(_adam(beta2=-0.1)) == L.L4D_EINVAL
    assert _adam_rc(_adam(eps=-1e-8)) == L.L4D_EINVAL
    assert _adam_rc(_adam(lr=float("nan"))) == L.L4D_EINVAL
    assert _adam_rc(_adam(grad_scale=float("inf"))) == L.L4D_EINVAL
    assert _adam_rc(_adam(), n=-1) == L.L4D_EINVAL
    assert L.lib().l4d_adam_step(None, 4, FAKE_BASE, FAKE_BASE, FAKE_BASE, FAKE_BASE, FAKE_BASE, None) == L.L4D_EINVAL
    base = [FAKE_BASE + (i << 20) for i in range(5)]
    for i in range(5):
        p = list(base)
        p[i] = None
        assert _adam_rc(_adam(), ptrs=p) == L.L4D_EINVAL
        p[i] = base[i] + (4 if i < 4 else 2)          # misaligned
        assert _adam_rc(_adam(), ptrs=p) == L.L4D_EINVAL
    # overlapping arrays: m starts inside the master's 4n bytes
    p = list(base)
    p[2] = base[1] + 2048
    assert _adam_rc(_adam(), n=1024, ptrs=p) == L.L4D_EINVAL
    assert "overlap" in L.lib().l4d_last_error().decode()
    # an empty shard is accepted and launches nothing
    assert _adam_rc(_adam(), n=0) == L.L4D_OK


def test_adam_step_rejects_oversized_shard():
    assert _adam_rc(_adam(), n=(1 << 33) + 4) == L.L4D_EINVAL
    assert "too large" in L.lib().l4d_last_error().decode()


def test_mem_fit_equals_the_oracle_on_every_printed_run():
    gold = os.path.join(os.path.dirname(__file__), "golden")
    names = {"fits": "green", "near_limit": "yellow", "oom": "red"}
    arch = {"llama-3.1-8b": (4096, 32, 8, 14336, 32, 128256), "llama-3.1-70b": (8192, 64, 8, 28672, 80, 128256)}
    n = 0
    for fn in ("paper_oom_outcomes.json", "paper_memory_tables.json"):
        with open(os.path.join(gold, fn)) as f:
            for c in json.load(f)["cells"]:
                h, a, k, ffn, layers, v = arch[c["model"]]
                d = c["n_gpus"] // (c["tp"] * c["cp"] * c["pp"])
                m = L.make_model(hidden=h, n_heads=a, n_kv_heads=k, ffn=ffn, n_layers=layers, vocab=v)
                p = L.make_parallel(seq=c["seq"], micro_batch=c["mbs"], tp=c["tp"], cp=c["cp"], pp=c["pp"], dp=d)
                est = L.mem_estimate(m, p)
                got = L.mem_fit(est, c["gpu_mem_gb"] << 30)
                want = M.oom_class(M.estimate(h, a, k, ffn, layers, v, s=c["seq"], b=c["mbs"], t=c["tp"],
                                              c=c["cp"], p=c["pp"], d=d)["total"], c["gpu_mem_gb"] << 30)
                assert names[got] == want == c["colour"], c
                n += 1
    assert n == 908
    gib = 1 << 30
    base = L.mem_estimate(*model_par(TINY))
    for total, fit in ((32 * gib, "fits"), (32 * gib + 1, "near_limit"), (40 * gib, "near_limit"),
                       (40 * gib + 1, "oom"), ((1 << 64) - 1, "oom")):
        assert L.mem_fit(dict(base, total_bytes=total), 40 * gib) == fit
    with pytest.raises(L.L4DError):
        L.mem_fit(base, 0)


def test_lm_head_noalloc_rejects_oversized_problems_before_touching_the_device():
    # 2048 tokens x a 32064-wide shard need 131 MB of logits: more than the 64 MiB static workspace
    lib = L.lib()
    f = C.c_void_p(FAKE_BASE)
    rc = lib.lm_head_xent_noalloc(2048, 4096, 32064, 0, f, f, f, f, f, 1.0, f, f, f, None)
    assert rc == L.L4D_EINVAL
    assert "static scratch" in lib.l4d_last_error().decode()
