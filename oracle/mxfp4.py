"""CPU oracle for the MoE layer with MXFP4 expert weights (float64, NumPy).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call this
module: only the tests, the smoke check and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP library and never imports it.

The paper serves GPT-OSS-120B with its expert weights in mxfp4 (Evaluation,
"Models"); the layer is otherwise the one in ``moe_oracle`` (standard top-k
gating, SwiGLU experts).  The paper does not define the format, so this module
follows the published OCP Microscaling (MX) specification, v1.0:

* an MXFP4 block is 32 elements that share one scale X;
* each element is FP4 E2M1: a sign bit, a 2-bit exponent with bias 1 and a
  1-bit mantissa; exponent 0 encodes the subnormals 0 and 0.5; there is no
  infinity or NaN, and the largest magnitude is 6;
* the scale is E8M0: an unsigned 8-bit exponent, X = 2^(code - 127); code 255
  is NaN;
* the value of element i is X * P_i.

Readings where the paper and the format leave a choice (listed in the design
notes):

* blocks run along the reduction axis of each weight matrix ([out, in]
  storage, 32 consecutive ``in`` values per block), as in the GPT-OSS
  checkpoints;
* two elements share a byte, the one with the lower index in the low nibble;
* weights are dequantized exactly (float64 holds every X * P_i) and the layer
  then runs in float64, like the bf16 oracle.

Inputs: each expert matrix is a pair ``(codes, scales)``: codes uint8
[E, R, K/2] (two elements a byte), scales uint8 [E, R, K/32].

Pins (CPU test suite): the E2M1 table printed in the OCP specification, the
E8M0 decoding of PyTorch's float8_e8m0fnu, hand-worked bytes, per-block scale
placement, nearest-grid-point consistency with an independent quantizer, and
the bf16 oracle on weights that bf16 represents exactly.
"""
from __future__ import annotations

import numpy as np

from oracle import moe_oracle

BLOCK = 32  # elements per MX block


# --------------------------------------------------------------------------
# Element and scale decoding
# --------------------------------------------------------------------------

def e2m1_decode(codes: np.ndarray) -> np.ndarray:
    """FP4 E2M1 code (low 4 bits) -> float64 value, from the bit fields.

    sign = bit 3, exponent field e = bits 2..1 (bias 1), mantissa m = bit 0:
    e > 0 is the normal number 2^(e - 1) * (1 + m / 2); e = 0 is the subnormal
    2^(1 - 1) * (m / 2).
    """
    c = np.asarray(codes).astype(np.int64) & 0xF
    sign = np.where((c >> 3) & 1, -1.0, 1.0)
    e = (c >> 1) & 3
    m = (c & 1).astype(np.float64)
    normal = np.ldexp(1.0 + m / 2.0, (e - 1).astype(np.int32))
    sub = m / 2.0
    return sign * np.where(e > 0, normal, sub)


def e8m0_decode(codes: np.ndarray) -> np.ndarray:
    """E8M0 scale code -> float64 2^(code - 127); code 255 is NaN."""
    c = np.asarray(codes).astype(np.int64)
    x = np.ldexp(1.0, (c - 127).astype(np.int32))
    return np.where(c == 255, np.nan, x)


def dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """(codes [..., K/2], scales [..., K/32]) -> float64 weights [..., K].

    Element k of a row sits in byte k // 2 (low nibble for even k, high nibble
    for odd k) and takes the scale of its block, k // 32.
    """
    b = np.asarray(codes, dtype=np.uint8)
    K = b.shape[-1] * 2
    nib = np.empty(b.shape[:-1] + (K,), dtype=np.uint8)
    nib[..., 0::2] = b & 0xF
    nib[..., 1::2] = b >> 4
    vals = e2m1_decode(nib)
    x = e8m0_decode(scales)
    assert x.shape[-1] * BLOCK == K, "one scale per 32 elements"
    return vals * np.repeat(x, BLOCK, axis=-1)


# --------------------------------------------------------------------------
# Expert FFN and layer
# --------------------------------------------------------------------------

def expert_ffn(x: np.ndarray, q1, q3, q2, ids: np.ndarray, buckets: dict) -> np.ndarray:
    """Expert outputs per slot, float64 [T*k, H], from MXFP4 weights.

    For the slot of pair (t, e): y = W2_e (silu(W1_e x_t) * (W3_e x_t)) with
    each W the dequantized matrix [out, in]; only union experts are touched.
    """
    T, H = x.shape
    x64 = np.asarray(x, dtype=np.float64)
    y = np.zeros((T * ids.shape[1], H), dtype=np.float64)
    offs = buckets["offsets"]
    perm = buckets["perm_token"]
    for e in buckets["union_ids"]:
        e = int(e)
        s0, s1 = int(offs[e]), int(offs[e + 1])
        xe = x64[perm[s0:s1]]
        W1 = dequantize(q1[0][e], q1[1][e])    # [I, H]
        W3 = dequantize(q3[0][e], q3[1][e])    # [I, H]
        W2 = dequantize(q2[0][e], q2[1][e])    # [H, I]
        g = xe @ W1.T
        v = xe @ W3.T
        h = moe_oracle.silu(g) * v
        y[s0:s1] = h @ W2.T
    return y


def moe_layer_routed(x, ids, weights, q1, q3, q2, E: int) -> dict:
    """The layer from given routing: buckets, union, slot outputs, output."""
    b = moe_oracle.bucket(ids, E)
    y = expert_ffn(x, q1, q3, q2, ids, b)
    out = moe_oracle.combine(y, b["pair_pos"], weights)
    return {**b, "y_slots": y, "out": out}


def moe_layer(x, w_gate, q1, q3, q2, k: int) -> dict:
    """The gate-routed layer with MXFP4 experts (the gate stays fp32)."""
    logits = moe_oracle.gate_logits(x, w_gate)
    ids = moe_oracle.select_experts(logits, k)
    w = moe_oracle.routing_weights(logits, ids)
    res = moe_layer_routed(x, ids, w, q1, q3, q2, E=w_gate.shape[0])
    return {"logits": logits, "ids": ids, "weights": w,
            "gaps": moe_oracle.selection_gaps(logits, k), **res}
