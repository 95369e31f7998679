"""The benchmark's work accounting, pinned on the CPU.

bench.py prices a layer step at 3 x (forward GEMM flops + unmasked attention
flops) and each kernel launch at its algorithmic flops or bytes.  These tests
tie those counts to the paper's parameter count (Eqs. 1-3: a layer's matrix
parameters on one TP rank, Sec. 3.1.2) and to closed forms of the causal
pair count, and check the staleness rule of the measured-traffic lookup.
"""
import hashlib
import os

import pytest

import bench
import workloads as W
from oracle import memory as OM

LAYERS = [W.TINY, W.LLAMA2_7B, W.LLAMA3_8B_TP2CP2, W.LLAMA3_70B_TP8]


@pytest.mark.parametrize("w", LAYERS, ids=lambda w: w.name)
def test_forward_gemm_flops_are_two_flops_per_matrix_parameter_and_token(w):
    # every matrix parameter of the rank's layer shard meets every local token once in the forward
    _, gemm_fwd, _ = bench.layer_flops(w)
    matrix_params = OM.layer_params(w.hidden, w.n_heads, w.n_kv_heads, w.ffn, w.tp) - 2 * w.hidden
    assert matrix_params.denominator == 1
    assert gemm_fwd == 2 * w.micro_batch * w.s_c * int(matrix_params)


@pytest.mark.parametrize("w", LAYERS, ids=lambda w: w.name)
def test_causal_pairs_have_closed_forms(w):
    s = w.seq
    if w.cp == 1:
        assert bench.attn_pairs(w) == s * (s + 1) // 2
    else:
        # the balanced chunk layout gives every CP rank the same share of the causal pairs
        assert bench.attn_pairs(w) * w.cp == s * (s + 1) // 2
        other = w.replace(cp_rank=(w.cp_rank + 1) % w.cp)
        assert bench.attn_pairs(other) == bench.attn_pairs(w)


@pytest.mark.parametrize("w", LAYERS, ids=lambda w: w.name)
def test_backward_gemms_cost_twice_the_forward(w):
    work = bench.kernel_work(w)
    fwd = sum(work[k][1] for k in ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down"))
    bwd = sum(v[1] for k, v in work.items() if k.startswith("gemm_") and k.endswith(("_dx", "_dw")))
    assert bwd == 2 * fwd
    total, gemm_fwd, attn_fwd = bench.layer_flops(w)
    assert fwd == gemm_fwd and total == 3 * (gemm_fwd + attn_fwd)
    assert work["attn_bwd_dkdv"][1] + work["attn_bwd_dq"][1] == 2 * attn_fwd


def test_headline_shard_flops():
    # Llama-3-70B at TP8, sequence 8192: the number the benchmark divides by its step time
    total, _, _ = bench.layer_flops(W.LLAMA3_70B_TP8)
    assert total == 5_669_407_162_368


def test_measured_traffic_is_dropped_once_the_source_changes(tmp_path):
    src = os.path.join(bench.ROOT, "paper_2411_06465_amd", "csrc", "gemm.hip")
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    f = tmp_path / "traffic.txt"
    f.write_text(f"# header\ntraffic gemm_gate_up_dw 123456 gemm.hip {sha}\n"
                 f"traffic gemm_down_dw 777 gemm.hip {'0' * 16}\n")
    assert bench.measured_traffic("gemm_gate_up_dw", str(f)) == 123456
    assert bench.measured_traffic("gemm_down_dw", str(f)) is None      # measured on another version
    assert bench.measured_traffic("gemm_qkv", str(f)) is None          # not measured
    assert bench.measured_traffic("gemm_qkv", str(tmp_path / "absent.txt")) is None
