"""The oracle still reproduces the frozen tiny-layer answer exactly."""
import json
import os

import numpy as np

from oracle import moe_oracle
from paper_2607_00466_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tiny_layer_seed0.json")


def test_tiny_golden():
    g = json.load(open(GOLDEN))
    s = synth.SHAPES["tiny"]
    x = synth.hidden_states(8, s.H, seed=0)
    wg = synth.gate_weights(s, seed=0)
    w1, w3, w2 = (synth.bf16_bits(t) for t in synth.expert_weights(s, seed=0))
    r = moe_oracle.moe_layer(x, wg, w1, w3, w2, s.K)
    for key in ("ids", "counts", "offsets", "perm_token", "pair_pos", "union_ids"):
        assert np.array_equal(np.asarray(g[key]), r[key]), key
    assert g["union_size"] == r["union_size"]
    np.testing.assert_allclose(r["weights"], g["weights"], rtol=1e-15, atol=0)
    np.testing.assert_allclose(r["out"], g["out"], rtol=1e-14, atol=1e-18)
