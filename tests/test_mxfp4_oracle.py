"""The MXFP4 oracle against its pins, and the pins against planted mistakes.

Pins (none of them re-types the oracle's own decoding):
- the FP4 E2M1 value table printed in the OCP Microscaling specification;
- E8M0 decoding against PyTorch's float8_e8m0fnu conversion (a library routine);
- hand-worked bytes for the nibble order and block scaling;
- per-block scale placement with a distinct scale per block;
- consistency with the generator's quantizer: every dequantized value is the
  grid point nearest to the fp32 draw (brute force over all 16 codes) unless
  the draw saturates;
- the expert FFN against the bf16 oracle on MXFP4 weights that bf16 holds
  exactly (every MXFP4 value with a scale in range is a bf16 number);
- the dense brute force of the bf16 path on the same weights.
"""
import importlib.util
import os

import numpy as np
import pytest
import torch

from oracle import bruteforce, moe_oracle
from oracle import mxfp4 as mx_oracle
from paper_2607_00466_amd import synth

SRC = os.path.join(os.path.dirname(mx_oracle.__file__), "mxfp4.py")

# OCP Microscaling Formats (MX) v1.0, FP4 E2M1 encodings 0000 .. 1111.
SPEC_E2M1 = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0,
             -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]


def _bf16_bits_exact(w: np.ndarray) -> np.ndarray:
    """float64 values that bf16 holds exactly -> bf16 bit patterns (checked)."""
    f = w.astype(np.float32)
    assert np.array_equal(f.astype(np.float64), w)
    bits = f.view(np.uint32)
    assert not (bits & 0xFFFF).any(), "value not representable in bf16"
    return (bits >> 16).astype(np.uint16)


def _small_layer(T=12, E=6, K=2, H=64, I=96, seed=4):
    sh = synth.LayerShape("mx_small", E=E, K=K, H=H, I=I)
    q = synth.mxfp4_expert_weights(sh, seed=seed)
    q = {k: (c.numpy(), s.numpy()) for k, (c, s) in q.items()}
    x = synth.hidden_states(T, H, seed=seed)
    ids, w, _ = synth.controlled_routing(T, E, K, U=E, seed=seed)
    return sh, q, x, ids, w


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def pin_e2m1_spec_table(O):
    got = O.e2m1_decode(np.arange(16))
    assert got.tolist() == SPEC_E2M1
    assert np.array_equal(np.signbit(got), np.arange(16) >= 8)


def pin_e8m0_matches_torch(O):
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    got = O.e8m0_decode(codes)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


def pin_hand_worked_bytes(O):
    # byte 0x21: element 0 = code 1 (0.5), element 1 = code 2 (1.0); 0xF9:
    # code 9 (-0.5), code 15 (-6); scale code 128 = 2, then 125 = 1/4
    codes = np.zeros((1, 32), np.uint8)
    codes[0, 0] = 0x21
    codes[0, 1] = 0xF9
    codes[0, 16] = 0x7E        # block 1: element 32 = code 14 (-4), 33 = code 7 (6)
    scales = np.array([[128, 125]], np.uint8)
    w = O.dequantize(codes, scales)
    assert w.shape == (1, 64)
    assert w[0, :4].tolist() == [1.0, 2.0, -1.0, -12.0]
    assert w[0, 32:34].tolist() == [-1.0, 1.5]
    assert not w[0, 4:32].any() and not w[0, 34:].any()


def pin_block_scale_placement(O):
    rng = np.random.default_rng(1)
    R, K = 3, 160
    codes = rng.integers(0, 256, (R, K // 2), dtype=np.uint8)
    scales = rng.integers(100, 140, (R, K // 32), dtype=np.uint8)
    w = O.dequantize(codes, scales)
    for r in range(R):
        for k in range(K):
            byte = int(codes[r, k // 2])
            nib = byte & 0xF if k % 2 == 0 else byte >> 4
            assert w[r, k] == SPEC_E2M1[nib] * 2.0 ** (int(scales[r, k // 32]) - 127)


def pin_nearest_grid_point(O):
    sh = synth.LayerShape("mx_pin", E=1, K=1, H=256, I=64)
    g = torch.Generator()
    g.manual_seed(7)
    draw = torch.randn((64, 256), generator=g) * synth.WEIGHT_STD
    c, s = synth._mxfp4_quantize(draw)
    w = O.dequantize(c.numpy(), s.numpy())
    X = 2.0 ** (s.numpy().astype(np.float64) - 127)
    Xk = np.repeat(X, 32, axis=-1)
    v = draw.numpy().astype(np.float64) / Xk
    grid = np.array(SPEC_E2M1)
    dist = np.abs(v[..., None] - grid)
    best = dist.min(axis=-1)
    got = w / Xk
    # the dequantized value is one of the nearest grid points (ties either way)
    assert np.allclose(np.abs(v - got), best, rtol=0, atol=1e-12)
    assert np.abs(got).max() <= 6.0
    # the shared exponent puts each block's largest value in [4, 8)
    amax = np.abs(v).reshape(64, 8, 32).max(-1)
    assert ((amax >= 4) & (amax < 8)).all()
    del sh


def pin_ffn_matches_bf16_oracle(O):
    sh, q, x, ids, _ = _small_layer()
    b = moe_oracle.bucket(ids, sh.E)
    got = O.expert_ffn(x, q["w1"], q["w3"], q["w2"], ids, b)
    bits = {k: _bf16_bits_exact(O.dequantize(*q[k])) for k in q}
    # bf16 patterns built from the spec table directly, not from the oracle
    for k in q:
        c, s = q[k]
        nib = np.stack([c & 0xF, c >> 4], axis=-1).reshape(c.shape[:-1] + (c.shape[-1] * 2,))
        ref = np.array(SPEC_E2M1)[nib] * np.repeat(2.0 ** (s.astype(np.float64) - 127), 32, axis=-1)
        assert np.array_equal(moe_oracle.widen_bf16(bits[k]), ref)
    ref = moe_oracle.expert_ffn(x, bits["w1"], bits["w3"], bits["w2"], ids, b)
    assert np.array_equal(got, ref)


def pin_layer_matches_bruteforce(O):
    sh, q, x, _, _ = _small_layer(T=9, E=5, K=3, seed=6)
    g = synth.gate_weights(sh, seed=6)
    res = O.moe_layer(x, g, q["w1"], q["w3"], q["w2"], sh.K)
    bits = {k: _bf16_bits_exact(O.dequantize(*q[k])) for k in q}
    bf = bruteforce.dense_layer(x, g, bits["w1"], bits["w3"], bits["w2"], sh.K)
    assert np.array_equal(res["ids"], bf["ids"])
    assert np.allclose(res["out"], bf["out"], rtol=1e-12, atol=1e-12)


ALL_PINS = [pin_e2m1_spec_table, pin_e8m0_matches_torch, pin_hand_worked_bytes,
            pin_block_scale_placement, pin_nearest_grid_point, pin_ffn_matches_bf16_oracle,
            pin_layer_matches_bruteforce]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(mx_oracle)


def _mutant(old: str, new: str):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    spec = importlib.util.spec_from_loader("mxfp4_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src.replace(old, new), "mxfp4_mutant", "exec"), mod.__dict__)
    return mod


# One plausible mistake per part of the oracle; each must be caught by some pin.
MUTATIONS = {
    "nibbles_swapped": ("nib[..., 0::2] = b & 0xF", "nib[..., 0::2] = b >> 4"),
    "exponent_bias_0": ("(e - 1).astype(np.int32)", "e.astype(np.int32)"),
    "subnormal_is_one": ("sub = m / 2.0", "sub = m"),
    "sign_dropped": ("sign = np.where((c >> 3) & 1, -1.0, 1.0)", "sign = 1.0"),
    "mantissa_quarter": ("(1.0 + m / 2.0", "(1.0 + m / 4.0"),
    "scale_bias_128": ("(c - 127).astype(np.int32)", "(c - 128).astype(np.int32)"),
    "scale_nan_ignored": ("np.where(c == 255, np.nan, x)", "x"),
    "scales_tiled": ("np.repeat(x, BLOCK, axis=-1)", "np.tile(x, BLOCK)"),
    "w1_w3_swapped": ("g = xe @ W1.T", "g = xe @ W3.T"),
    "down_transposed": ("y[s0:s1] = h @ W2.T", "y[s0:s1] = h @ W2[:, ::-1].T"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name):
    mod = _mutant(*MUTATIONS[name])
    caught = []
    for pin in ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mod)
        except Exception:  # an assertion or a crash both mean the pin caught it
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {name}"
