"""The CPU oracle against its pins, and the pins against planted mistakes."""
import importlib.util
import os

import numpy as np
import pytest

from oracle import moe_oracle
from tests import oracle_pins

ORACLE_SRC = os.path.join(os.path.dirname(moe_oracle.__file__), "moe_oracle.py")


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(moe_oracle)


def _mutant(old: str, new: str):
    src = open(ORACLE_SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    spec = importlib.util.spec_from_loader("oracle_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


# One plausible mistake per part of the oracle; each must be caught by some pin.
MUTATIONS = {
    "tie_to_higher_id": ("logits[t, e] > logits[t, best]", "logits[t, e] >= logits[t, best]"),
    "no_renormalise": ("w[t] = sel / np.sum(sel)", "w[t] = sel"),
    "softmax_sign": ("p = np.exp(logits[t] - m)", "p = np.exp(m - logits[t])"),
    "silu_is_sigmoid": ("return z / (1.0 + np.exp(-z))", "return 1.0 / (1.0 + np.exp(-z))"),
    "swiglu_swapped": ("h = silu(g) * v", "h = silu(v) * g"),
    "w1_dropped": ("g = xe @ W1.T", "g = xe @ W3.T"),
    "down_index_reversed": ("y[s0:s1] = h @ W2.T", "y[s0:s1] = h @ W2[:, ::-1].T"),
    "combine_unweighted": ("out[t] += float(weights[t, j]) * y_slots[int(pair_pos[t, j])]",
                           "out[t] += y_slots[int(pair_pos[t, j])]"),
    "bucket_tokens_descending": ("for t in range(T):  # ascending t", "for t in reversed(range(T)):  #"),
    "gate_term_dropped": ("return x64 @ g64.T", "return x64[:, :-1] @ g64[:, :-1].T"),
    "bf16_shift": ("<< np.uint32(16)", "<< np.uint32(15)"),
    "union_all_experts": ("if counts[e] > 0]", "if counts[e] >= 0]"),
    "gap_off_by_one": ("s[:, k - 1] - s[:, k]", "s[:, k - 1] - s[:, k - 1]"),
    "offsets_shifted": ("offsets[e + 1] = offsets[e] + counts[e]", "offsets[e + 1] = counts[e]"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name):
    mod = _mutant(*MUTATIONS[name])
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mod)
        except Exception:  # an assertion or a crash both mean the pin caught it
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {name}"
