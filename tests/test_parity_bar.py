"""The parity bar itself (CPU): a single rounding-boundary flip propagated
through a sum passes, a corrupted block or a systematic error fails."""
import numpy as np

from gpu_common import check
from oracle.bf16 import round_bf16


def test_bar_accepts_rounding_flips_and_rejects_block_errors():
    rng = np.random.default_rng(0)
    h1 = round_bf16(rng.standard_normal((64, 512)) * 3)
    f = round_bf16(rng.standard_normal((64, 512)))
    ref = round_bf16(h1 + f)
    # one operand rounds one step the other way in a few elements: the sum moves by that step
    h1_flip = h1.copy()
    idx = rng.choice(h1.size, 30, replace=False)
    step = np.ldexp(1.0, (np.floor(np.log2(np.abs(h1.flat[idx]))) - 7).astype(int))
    h1_flip.flat[idx] += step
    assert check("flip", round_bf16(h1_flip + f), ref)
    # a block of 8 x 64 wrong by its own size
    bad = ref.copy()
    bad[8:16, 64:128] *= -1
    assert not check("block", bad, ref)
    # a systematic 1% scale error
    assert not check("scale", round_bf16(ref * 1.01), ref)
    # fp32 outputs: Frobenius only
    assert check("fp32", ref * (1 + 1e-3), ref, bf16=False)
