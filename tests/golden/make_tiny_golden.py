"""Write tests/golden/tiny_layer_seed0.json from the CPU oracle.

The tiny workload (E=16 experts, top-2, hidden 256, expert intermediate 128,
8 tokens, seed 0, gate-routed) run through the float64 oracle only.  The file
freezes the oracle's answer so that a later change to its arithmetic shows up
as a failing test and has to be justified.  Run from the repository root:

    python tests/golden/make_tiny_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import moe_oracle  # noqa: E402
from paper_2607_00466_amd import synth  # noqa: E402


def main() -> None:
    s = synth.SHAPES["tiny"]
    x = synth.hidden_states(8, s.H, seed=0)
    wg = synth.gate_weights(s, seed=0)
    w1, w3, w2 = (synth.bf16_bits(t) for t in synth.expert_weights(s, seed=0))
    r = moe_oracle.moe_layer(x, wg, w1, w3, w2, s.K)
    doc = {
        "workload": "tiny MoE layer: E=16, top-2, H=256, I=128, T=8, seed 0, gate-routed",
        "source": "CPU float64 oracle (oracle/moe_oracle.py) on synth inputs",
        "ids": r["ids"].tolist(),
        "weights": [[float(v) for v in row] for row in r["weights"]],
        "gaps": [float(v) for v in r["gaps"]],
        "counts": r["counts"].tolist(),
        "offsets": r["offsets"].tolist(),
        "perm_token": r["perm_token"].tolist(),
        "pair_pos": r["pair_pos"].tolist(),
        "union_ids": r["union_ids"].tolist(),
        "union_size": int(r["union_size"]),
        "out": [[float(v) for v in row] for row in r["out"]],
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_layer_seed0.json")
    with open(path, "w") as f:
        json.dump(doc, f, separators=(",", ":"))
        f.write("\n")
    print("wrote", path)


if __name__ == "__main__":
    main()
