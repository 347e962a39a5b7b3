"""CPU oracle for one batched-decode MoE layer (float64, NumPy).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call this
module: only the tests, the smoke check and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP library and never imports it.

What it computes is the plain definition of the layer that ELDR leaves
untouched (Introduction and Related Work: the router changes only which decode
worker serves a request, so expert selections and outputs are those of
standard top-k gating).  The layer (Background, Mixture-of-Experts LLMs) is an
MoE gate that scores every expert from the token's hidden state (Introduction,
footnote on the MoE gate) followed by the expert FFNs of the k experts the
token selects; only the discrete top-k fetch an expert, the remaining scores
are computed and discarded (Design, Signature Design, "discrete, not
continuous").  The step cost is the union of distinct experts the batch
activates (Motivation, Active Expert Count Drives MoE Decode Latency); that
union and the per-expert buckets are computed here as plain sets and counts.

Readings where the paper is silent (each is listed in the design notes):

* softmax over all E experts, then top-k, then renormalise over the k chosen;
* selection compares logits, ties go to the lower expert id;
* SwiGLU FFN ``W2 (silu(W1 x) * (W3 x))`` with no bias, clamp or scaling;
* no expert capacity, dropping, shared expert or gate bias;
* within a bucket tokens are in ascending token order; the union is ascending.

Inputs: x [T,H] fp32, w_gate [E,H] fp32, expert weights as raw bf16 bit
patterns (uint16) w1/w3 [E,I,H] and w2 [E,H,I].  All arithmetic is float64 on
the exact input values (bf16 and fp32 widen exactly).

Pins: every function here is checked, in the CPU test suite, against something
other than itself (dense brute force, library routines, closed forms, special
cases and invariants); no function is "parity unpinned".
"""
from __future__ import annotations

import numpy as np


# --------------------------------------------------------------------------
# Inputs
# --------------------------------------------------------------------------

def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values.

    A bf16 number is the upper 16 bits of an IEEE binary32 number, so shifting
    the pattern into the high half of a 32-bit word gives the same value as a
    float32, which widens exactly to float64.
    """
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Gate: scores, selection, weights
# --------------------------------------------------------------------------

def gate_logits(x: np.ndarray, w_gate: np.ndarray) -> np.ndarray:
    """Gate scores l[t, e] = sum_h x[t, h] * w_gate[e, h], float64 [T, E].

    The MoE gate scores every expert from the token's hidden state
    (Introduction; Background, Mixture-of-Experts LLMs).
    """
    x64 = np.asarray(x, dtype=np.float64)
    g64 = np.asarray(w_gate, dtype=np.float64)
    return x64 @ g64.T


def select_experts(logits: np.ndarray, k: int) -> np.ndarray:
    """Each token's k selected experts, int32 [T, k].

    Listed in selection order: larger logit first; between equal logits the
    lower expert id first.  Selection is by logit (softmax is monotone, so this
    is the same set as top-k of the probabilities without rounding effects).
    """
    T, E = logits.shape
    if not 1 <= k <= E:
        raise ValueError("need 1 <= k <= E")
    ids = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        taken = np.zeros(E, dtype=bool)
        for j in range(k):
            best = -1
            for e in range(E):
                if taken[e]:
                    continue
                if best < 0 or logits[t, e] > logits[t, best]:
                    best = e  # strict '>' keeps the lower id on a tie
            taken[best] = True
            ids[t, j] = best
    return ids


def routing_weights(logits: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Combine weights [T, k] float64: softmax over all E, renormalised over the k picks.

    p = softmax(l_t) over every expert (the gate's probability mass spans all E
    experts; Design, Signature Design), then w_tj = p[ids_tj] / sum_j' p[ids_tj'].
    """
    T, E = logits.shape
    k = ids.shape[1]
    w = np.empty((T, k), dtype=np.float64)
    for t in range(T):
        m = np.max(logits[t])
        p = np.exp(logits[t] - m)
        p = p / np.sum(p)
        sel = p[ids[t]]
        w[t] = sel / np.sum(sel)
    return w


def selection_gaps(logits: np.ndarray, k: int) -> np.ndarray:
    """Per-token margin of the selection, float64 [T].

    gap_t = (k-th largest logit) - ((k+1)-th largest logit); +inf when k == E
    (nothing is left out).  A token whose gap is below the near-tie threshold
    may legitimately select a different set under a different rounding order.
    """
    T, E = logits.shape
    if k == E:
        return np.full(T, np.inf)
    s = -np.sort(-logits, axis=1)
    return s[:, k - 1] - s[:, k]


# --------------------------------------------------------------------------
# Buckets and the distinct-expert union
# --------------------------------------------------------------------------

def bucket(ids: np.ndarray, E: int) -> dict[str, np.ndarray | int]:
    """Group (token, expert) pairs by expert; the distinct-expert union.

    counts[e]      number of tokens that selected e
    offsets[e]     sum of counts[e'] for e' < e  (offsets[E] = T*k)
    perm_token[s]  token of slot s: experts ascending, tokens ascending within
    pair_pos[t,j]  slot of the pair (t, ids[t, j])
    union_ids      experts with counts > 0, ascending; union_size = len

    The union is the set of distinct experts the batch activates, whose
    weights a decode step must fetch (Motivation, Active Expert Count Drives
    MoE Decode Latency).
    """
    T, k = ids.shape
    counts = np.zeros(E, dtype=np.int64)
    for t in range(T):
        for j in range(k):
            counts[int(ids[t, j])] += 1
    offsets = np.zeros(E + 1, dtype=np.int64)
    for e in range(E):
        offsets[e + 1] = offsets[e] + counts[e]
    perm_token = np.empty(T * k, dtype=np.int64)
    pair_pos = np.empty((T, k), dtype=np.int64)
    fill = offsets[:E].copy()
    for t in range(T):  # ascending t, so each bucket lists its tokens in order
        for j in range(k):
            e = int(ids[t, j])
            perm_token[fill[e]] = t
            pair_pos[t, j] = fill[e]
            fill[e] += 1
    union_ids = np.array([e for e in range(E) if counts[e] > 0], dtype=np.int64)
    return {
        "counts": counts.astype(np.int32),
        "offsets": offsets.astype(np.int32),
        "perm_token": perm_token.astype(np.int32),
        "pair_pos": pair_pos.astype(np.int32),
        "union_ids": union_ids.astype(np.int32),
        "union_size": int(union_ids.size),
    }


# --------------------------------------------------------------------------
# Expert FFN and combine
# --------------------------------------------------------------------------

def silu(z: np.ndarray) -> np.ndarray:
    """silu(z) = z * sigmoid(z) = z / (1 + exp(-z))."""
    return z / (1.0 + np.exp(-z))


def expert_ffn(x: np.ndarray, w1: np.ndarray, w3: np.ndarray, w2: np.ndarray,
               ids: np.ndarray, buckets: dict) -> np.ndarray:
    """Expert outputs per slot, float64 [T*k, H].

    For the slot of pair (t, e): y = W2_e (silu(W1_e x_t) * (W3_e x_t)), each
    weight matrix stored [out, in].  Only experts in the union are touched,
    each once for all of its tokens (the step's cost model: every activated
    expert's weights, and nothing else; Motivation).
    """
    T, H = x.shape
    n_slots = T * ids.shape[1]
    x64 = np.asarray(x, dtype=np.float64)
    y = np.zeros((n_slots, H), dtype=np.float64)
    offs = buckets["offsets"]
    perm = buckets["perm_token"]
    for e in buckets["union_ids"]:
        e = int(e)
        s0, s1 = int(offs[e]), int(offs[e + 1])
        xe = x64[perm[s0:s1]]                  # [c_e, H]
        W1 = widen_bf16(w1[e])                 # [I, H]
        W3 = widen_bf16(w3[e])                 # [I, H]
        W2 = widen_bf16(w2[e])                 # [H, I]
        g = xe @ W1.T                          # [c_e, I]
        v = xe @ W3.T                          # [c_e, I]
        h = silu(g) * v                        # [c_e, I]
        y[s0:s1] = h @ W2.T                    # [c_e, H]
    return y


def combine(y_slots: np.ndarray, pair_pos: np.ndarray, weights: np.ndarray) -> np.ndarray:
    """out[t] = sum over j = 0..k-1 of weights[t, j] * y_slots[pair_pos[t, j]], float64 [T, H]."""
    T, k = pair_pos.shape
    out = np.zeros((T, y_slots.shape[1]), dtype=np.float64)
    for t in range(T):
        for j in range(k):
            out[t] += float(weights[t, j]) * y_slots[int(pair_pos[t, j])]
    return out


# --------------------------------------------------------------------------
# Whole layer
# --------------------------------------------------------------------------

def moe_layer_routed(x, ids, weights, w1, w3, w2, E: int) -> dict:
    """The layer from given routing (gate bypassed): buckets, union, slot outputs, output."""
    b = bucket(ids, E)
    y = expert_ffn(x, w1, w3, w2, ids, b)
    out = combine(y, b["pair_pos"], weights)
    return {**b, "y_slots": y, "out": out}


def moe_layer(x, w_gate, w1, w3, w2, k: int) -> dict:
    """The gate-routed layer: gate scores, top-k ids and weights, buckets, output."""
    logits = gate_logits(x, w_gate)
    ids = select_experts(logits, k)
    w = routing_weights(logits, ids)
    res = moe_layer_routed(x, ids, w, w1, w3, w2, E=w_gate.shape[0])
    return {"logits": logits, "ids": ids, "weights": w,
            "gaps": selection_gaps(logits, k), **res}
