"""The parity bar itself (CPU): rounding flips of a stored operand pass only
with that operand's allowance, contraction noise at the stated relative
tolerance passes, and a corrupted element, row or block, or a systematic
error, fails."""
import numpy as np

from gpu_common import bf16_ulp, check
from oracle.bf16 import round_bf16


def _residual_case(seed=0):
    rng = np.random.default_rng(seed)
    h1 = round_bf16(rng.standard_normal((64, 512)) * 8)
    f = round_bf16(-h1 + rng.standard_normal((64, 512)) * 0.3)    # y = h1 + f cancels to |y| ~ 0.3
    return rng, h1, f, round_bf16(h1 + f)


def test_flip_of_the_residual_operand_needs_its_allowance():
    rng, h1, f, ref = _residual_case()
    # h1 rounds one step the other way in a few elements: y moves by that step
    h1_flip = h1.copy()
    idx = rng.choice(h1.size, 30, replace=False)
    h1_flip.flat[idx] += bf16_ulp(h1.flat[idx])
    got = round_bf16(h1_flip + f)
    assert check("flip+allow", got, ref, allow=bf16_ulp(h1), contraction=False)
    # the flip is far larger than the result's own step: without the allowance it fails
    assert not check("flip-noallow", got, ref, contraction=False)


def test_contraction_noise_at_the_stated_tolerance_passes():
    # y = a W with every operand element off by 3e-3 relative (independent): each
    # output deviates by about 3e-3 of its row RMS (~6 here), also where y itself
    # is small, which the element bound without C does not admit
    rng = np.random.default_rng(4)
    a = rng.standard_normal((256, 1024)) * 10
    wt = rng.standard_normal((1024, 512)) * 0.02
    ref = round_bf16(a @ wt)
    got = round_bf16((a * (1 + 3e-3 * rng.standard_normal(a.shape))) @ wt)
    assert check("contraction", got, ref)
    assert not check("contraction-elementwise-bar", got, ref, contraction=False)


def test_bar_rejects_elements_blocks_rows_and_scale_errors():
    rng, h1, f, ref = _residual_case(1)
    allow = bf16_ulp(h1)
    bad = ref.copy()
    bad[8:16, 64:128] *= -1                      # a block wrong by its own size
    assert not check("block", bad, ref, allow=allow)
    row = ref.copy()
    row[5] += 0.01 * np.sign(row[5])             # one row off by 0.01: inside 2e-2 per element
    assert not check("row", row, ref, allow=allow)
    assert not check("scale", round_bf16(ref * 1.01), ref, allow=allow)
    one = ref.copy()
    one[3, 100] += 0.1                           # one element off by a third of the row RMS
    assert not check("element", one, ref, allow=allow)


def test_bar_catches_a_wrong_row_of_a_tiny_scale_tensor():
    # a gradient of magnitude ~1e-5: 2e-2 absolute is vacuous, the per-row bound is not
    rng = np.random.default_rng(2)
    ref = round_bf16(rng.standard_normal((256, 128)) * 1e-5)
    assert check("tiny-ok", ref, ref)
    bad = ref.copy()
    bad[17] = 0.0
    assert not check("tiny-row", bad, ref)


def test_a_value_rounding_into_the_next_binade_is_one_step_of_the_larger():
    ref = np.full((1, 4096), 7.9375)             # two bf16 steps (1/32 each) below 8
    got = ref.copy()
    got[0, 0] = 8.0                              # 8: one step of the binade it rounded into
    assert check("binade", got, ref, contraction=False)
    got[0, 0] = 8.0625                           # two steps of that binade
    assert not check("binade-2", got, ref, contraction=False)


def test_fp32_outputs_frobenius_rows_and_absolute_bound():
    rng = np.random.default_rng(3)
    ref = rng.standard_normal((128, 64))
    assert check("fp32", ref * (1 + 1e-3), ref, bf16=False)
    bad = ref.copy()
    bad[3] *= 1.1
    assert not check("fp32-row", bad, ref, bf16=False)
    lse = rng.standard_normal((4, 256)) + 8
    assert check("lse", lse + 1e-3, lse, bf16=False, abs_bound=2e-2)
    off = lse.copy()
    off[1, 7] += 0.05
    assert not check("lse-off", off, lse, bf16=False, abs_bound=2e-2)
