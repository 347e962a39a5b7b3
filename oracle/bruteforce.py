"""Dense brute force for the MoE layer: every expert on every token, then mask.

TEST INFRASTRUCTURE ONLY (same restriction as ``moe_oracle``).  This is a
second, independent route to the layer output used to pin the sparse oracle:
it computes FFN_e(x_t) for all (t, e) with einsum, builds the mask
M[t, e] = (renormalised top-k weight if e is selected by t, else 0), and sums
sum_e M[t, e] * FFN_e(x_t).  Because ELDR only changes placement, the layer
output must equal standard top-k gating (Introduction; Related Work), which is
exactly this masked dense sum.

Selection uses a stable argsort on the negated logits (a library routine; ties
keep the lower id) and the softmax is scipy's, so no code is shared with the
sparse oracle.
"""
from __future__ import annotations

import numpy as np
from scipy.special import softmax


def _widen(bits: np.ndarray) -> np.ndarray:
    # bf16 -> float32 by placing the 16 bits in the high half, then to float64.
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) * np.uint32(65536)
    return u32.view(np.float32).astype(np.float64)


def dense_topk_mask(logits: np.ndarray, k: int) -> tuple[np.ndarray, np.ndarray]:
    """Selected ids (as a sorted-by-rank array) and the dense [T, E] weight mask."""
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    probs = softmax(logits, axis=1)
    mask = np.zeros_like(logits)
    rows = np.arange(logits.shape[0])[:, None]
    sel = probs[rows, order]
    mask[rows, order] = sel / sel.sum(axis=1, keepdims=True)
    return order.astype(np.int32), mask


def dense_expert_outputs(x: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """FFN_e(x_t) for every token and every expert, float64 [T, E, H]."""
    x64 = np.asarray(x, dtype=np.float64)
    W1, W3, W2 = _widen(w1), _widen(w3), _widen(w2)
    g = np.einsum("th,eih->tei", x64, W1)
    v = np.einsum("th,eih->tei", x64, W3)
    h = g * (1.0 / (1.0 + np.exp(-g))) * v
    return np.einsum("tei,ehi->teh", h, W2)


def dense_layer(x, w_gate, w1, w3, w2, k: int) -> dict:
    """Gate-routed layer by brute force."""
    logits = np.einsum("th,eh->te", np.asarray(x, np.float64), np.asarray(w_gate, np.float64))
    ids, mask = dense_topk_mask(logits, k)
    Y = dense_expert_outputs(x, w1, w3, w2)
    return {"logits": logits, "ids": ids, "mask": mask, "out": np.einsum("te,teh->th", mask, Y)}


def dense_layer_routed(x, ids, weights, w1, w3, w2, E: int) -> np.ndarray:
    """Layer output from given routing by brute force: dense outputs times a scattered mask."""
    T = x.shape[0]
    mask = np.zeros((T, E), dtype=np.float64)
    for t in range(T):
        mask[t, ids[t]] += np.asarray(weights[t], dtype=np.float64)
    Y = dense_expert_outputs(x, w1, w3, w2)
    return np.einsum("te,teh->th", mask, Y)
