"""The GPU tests' gate checker on fabricated GPU outputs (CPU only).

The near-tie branch of `gpu_util.check_gate` accepts a selection that differs
from the oracle's only when it is valid: the top-k of the GPU's own logits
under the tie rule, swapping only experts inside the near-tie band of the
oracle's k-th logit.  These cases feed it outputs built by hand (no GPU, no
library call) and check that it accepts the valid pick and rejects the
invalid ones.
"""
import numpy as np
import pytest

from oracle import moe_oracle as O
from tests import gpu_util as G

E, H, K, T = 16, 256, 2, 8


def _inputs():
    # gate rows 5 and 9 differ by 2^-20 at position 200; x[200] = 0.1 makes the
    # two logits differ by 9.5e-8, below half an ulp of 2 in fp32
    wg = np.zeros((E, H), np.float32)
    wg[np.arange(E), np.arange(E)] = 1.0
    wg[9, 9], wg[9, 5], wg[9, 200] = 0.0, 1.0, 2.0 ** -20
    x = np.random.default_rng(1).uniform(-0.5, 0.5, (T, H)).astype(np.float32)
    x[:, 2], x[:, 5], x[:, 200] = 4.0, 2.0, 0.1
    return x, wg


def _gpu_like(x, wg, ids):
    """What the GPU returns: fp32 logits (here exact or one rounding), the given
    ids, and weights from those ids."""
    logits32 = (x.astype(np.float64) @ wg.astype(np.float64).T).astype(np.float32)
    w = O.routing_weights(O.gate_logits(x, wg), ids.astype(np.int64)).astype(np.float32)
    return {"logits": logits32, "ids": ids.astype(np.int32), "weights": w}


def test_valid_near_tie_pick_is_accepted():
    x, wg = _inputs()
    # fp32 sees logits 5 and 9 tied, so the lower id 5 is the valid pick; the
    # oracle (float64) picks 9
    ids = np.tile(np.array([2, 5]), (T, 1))
    assert set(O.select_experts(O.gate_logits(x, wg), K)[0].tolist()) == {2, 9}
    near = G.check_gate(_gpu_like(x, wg, ids), x, wg, K)
    assert near.all()


def test_pick_against_own_logits_is_rejected():
    x, wg = _inputs()
    g = _gpu_like(x, wg, np.tile(np.array([2, 9]), (T, 1)))
    # make the GPU's own logits prefer 5 strictly: picking 9 is then invalid
    g["logits"][:, 5] = np.nextafter(np.float32(2.0), np.float32(3.0))
    with pytest.raises(AssertionError, match="own logits"):
        G.check_gate(g, x, wg, K)


def test_swap_of_a_far_expert_is_rejected():
    x, wg = _inputs()
    ids = np.tile(np.array([2, 5]), (T, 1))
    ids[3] = [2, 11]  # logit 11 is far below the k-th logit (about 2)
    g = _gpu_like(x, wg, ids)
    # 11 as the GPU's own choice: its logit then strays from the oracle's too
    g["logits"][3, 11] = np.float32(3.0)
    with pytest.raises(AssertionError):
        G.check_gate(g, x, wg, K)


def test_wrong_set_on_a_clean_token_is_rejected():
    x, wg = _inputs()
    x[:, 200] = 0.0
    x[:, 5] = -3.0
    x[:, 7] = 2.0  # experts 2 and 7 lead by far: no near-tie
    ids = np.tile(np.array([2, 7]), (T, 1))
    assert not G.check_gate(_gpu_like(x, wg, ids), x, wg, K).any()
    ids[0] = [2, 4]
    with pytest.raises(AssertionError):
        G.check_gate(_gpu_like(x, wg, ids), x, wg, K)
