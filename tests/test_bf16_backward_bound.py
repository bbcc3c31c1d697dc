"""The 8-layer stage share's composed backward is held to 5e-2 of max|ref| on the GPU
instead of 2e-2.  This CPU test reproduces the reason from the oracle alone: rounding only
the forward activations that the bf16 path keeps (layer inputs, Q, K, V, O) to bf16, with
everything else exact, already moves this problem's gradients past 2e-2 (and stays below
5e-2)."""
import numpy as np
import pytest

from bf16_emulation import stage_share_prefix_gradients


def _rel(got, ref):
    return float(np.abs(got - ref).max() / np.abs(ref).max())


@pytest.mark.slow
def test_bf16_forward_rounding_alone_exceeds_the_2e2_bar():
    (dx_ref, g_ref), (dx_bf, g_bf) = stage_share_prefix_gradients(P=300, batch=4)
    e_dx = max(_rel(a, b) for a, b in zip(dx_bf, dx_ref))
    e_w = max(_rel(g_bf[l][k], g_ref[l][k]) for l in range(len(g_ref)) for k in g_ref[l]
              if g_ref[l][k] is not None)
    print(f"bf16-forward model vs exact oracle: dx {e_dx:.3e}, weight gradients {e_w:.3e}")
    assert max(e_dx, e_w) > 2e-2
    assert e_dx < 5e-2 and e_w < 5e-2
