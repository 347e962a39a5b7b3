"""Pins for the CPU oracle: checks against things other than the oracle itself.

Each ``pin_*`` function takes the oracle module (so a test can hand it a copy
with a planted mistake) and raises AssertionError when the oracle disagrees
with the mathematics or a library routine.  Pins never call the HIP library.
"""
from __future__ import annotations

import math

import numpy as np
import torch
from scipy.special import softmax

from oracle import bruteforce
from paper_2607_00466_amd import synth


def _bits(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of values that are exactly representable in bf16."""
    f = np.asarray(a, dtype=np.float32)
    u = f.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def _tiny_inputs(seed: int = 0, T: int = 8):
    s = synth.SHAPES["tiny"]
    x = synth.hidden_states(T, s.H, seed)
    wg = synth.gate_weights(s, seed)
    w1, w3, w2 = (synth.bf16_bits(t) for t in synth.expert_weights(s, seed))
    return s, x, wg, w1, w3, w2


def _small_routed(seed: int = 1, T: int = 12, E: int = 6, K: int = 3, H: int = 64, I: int = 32):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, H)).astype(np.float32)
    w = [synth.bf16_bits(torch.from_numpy(rng.normal(0, 0.05, sh).astype(np.float32)).to(torch.bfloat16))
         for sh in ((E, I, H), (E, I, H), (E, H, I))]
    ids = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    wts = rng.dirichlet(np.ones(K), size=T).astype(np.float32)
    return x, ids, wts, w[0], w[1], w[2], E


# ---------------------------------------------------------------- layer output

def pin_dense_bruteforce_gate_routed(O) -> None:
    """Sparse oracle == dense all-experts-then-mask on the tiny workload."""
    s, x, wg, w1, w3, w2 = _tiny_inputs()
    r = O.moe_layer(x, wg, w1, w3, w2, s.K)
    d = bruteforce.dense_layer(x, wg, w1, w3, w2, s.K)
    assert np.array_equal(np.sort(r["ids"], 1), np.sort(d["ids"], 1)), "selected sets differ"
    scale = np.abs(d["out"]).max()
    assert np.abs(r["out"] - d["out"]).max() <= 1e-12 * scale, "output differs from dense brute force"
    # the sparse weights, scattered densely, equal the brute-force mask
    dense_w = np.zeros_like(d["mask"])
    for t in range(r["ids"].shape[0]):
        dense_w[t, r["ids"][t]] = r["weights"][t]
    assert np.abs(dense_w - d["mask"]).max() <= 1e-15


def pin_dense_bruteforce_routed(O) -> None:
    """Gate-bypassed layer == dense brute force with the scattered routing weights."""
    x, ids, wts, w1, w3, w2, E = _small_routed()
    r = O.moe_layer_routed(x, ids, wts, w1, w3, w2, E)
    ref = bruteforce.dense_layer_routed(x, ids, wts, w1, w3, w2, E)
    assert np.abs(r["out"] - ref).max() <= 1e-12 * np.abs(ref).max()


def pin_single_expert_is_dense_swiglu(O) -> None:
    """E = 1, k = 1: the layer is one dense SwiGLU FFN, computed with torch's F.linear/F.silu."""
    rng = np.random.default_rng(3)
    T, H, I = 5, 48, 16
    x = rng.standard_normal((T, H)).astype(np.float32)
    Wt = [torch.from_numpy(rng.normal(0, 0.1, sh).astype(np.float32)).to(torch.bfloat16)
          for sh in ((1, I, H), (1, I, H), (1, H, I))]
    w1, w3, w2 = (synth.bf16_bits(t) for t in Wt)
    ids = np.zeros((T, 1), np.int32)
    wts = np.ones((T, 1), np.float32)
    r = O.moe_layer_routed(x, ids, wts, w1, w3, w2, 1)
    F = torch.nn.functional
    xt = torch.from_numpy(x).double()
    A, B, C = (t[0].double() for t in Wt)
    ref = F.linear(F.silu(F.linear(xt, A)) * F.linear(xt, B), C).numpy()
    assert np.abs(r["out"] - ref).max() <= 1e-12 * np.abs(ref).max()


def pin_zero_input(O) -> None:
    """x = 0: every logit is 0, so the first k ids win with weight 1/k; the output is 0."""
    s, x, wg, w1, w3, w2 = _tiny_inputs()
    x = np.zeros_like(x)
    r = O.moe_layer(x, wg, w1, w3, w2, s.K)
    assert np.array_equal(r["ids"], np.tile(np.arange(s.K, dtype=np.int32), (x.shape[0], 1)))
    assert np.all(r["weights"] == 1.0 / s.K)
    assert np.all(r["out"] == 0.0)
    assert r["union_size"] == s.K


def pin_down_projection_linear(O) -> None:
    """Doubling W2 (exact in bf16) doubles the output exactly; negating W3 negates it."""
    x, ids, wts, w1, w3, w2, E = _small_routed(seed=5)
    base = O.moe_layer_routed(x, ids, wts, w1, w3, w2, E)["out"]
    w2x2 = _bits(2.0 * O.widen_bf16(w2).astype(np.float32))
    assert np.array_equal(O.moe_layer_routed(x, ids, wts, w1, w3, w2x2, E)["out"], 2.0 * base)
    w3neg = w3 ^ np.uint16(0x8000)
    assert np.array_equal(O.moe_layer_routed(x, ids, wts, w1, w3neg, w2, E)["out"], -base)


def pin_closed_form_example(O) -> None:
    """A three-expert, two-dimensional layer whose output is worked out by hand.

    Gate rows e0 = (1, 0), e1 = (0, 1), e2 = (-1, 0); k = 2.
      token 0, x = (2, 1):   logits (2, 1, -2)  -> picks e0, e1;
                             weights e^2/(e^2+e) = e/(e+1) and 1/(e+1).
      token 1, x = (-1, -1): logits (-1, -1, 1) -> picks e2, then e0 (tie with
                             e1 at -1 goes to the lower id); weights
                             e/(e+1/e) = e^2/(e^2+1) and 1/(e^2+1).
    Experts (I = 1), rows are [out, in]:
      e0: W1 = (1, 0),  W3 = (0, 1),    W2 = (1, 2)^T
      e1: W1 = (0, 1),  W3 = (1, 0),    W2 = (-1, 0.5)^T
      e2: W1 = (1, 1),  W3 = (0.5, 0.5), W2 = (0.25, -1)^T
    With s(z) = z / (1 + e^-z):
      token 0: e0 gives h = s(2)*1, y = (h, 2h); e1 gives h = s(1)*2, y = (-h, h/2)
      token 1: e2 gives h = s(-2)*(-1), y = (h/4, -h); e0 gives h = s(-1)*(-1), y = (h, 2h)
    """
    e = math.e
    s = lambda z: z / (1.0 + math.exp(-z))  # noqa: E731  (the textbook definition)
    x = np.array([[2, 1], [-1, -1]], np.float32)
    wg = np.array([[1, 0], [0, 1], [-1, 0]], np.float32)
    w1 = _bits(np.array([[[1, 0]], [[0, 1]], [[1, 1]]], np.float32))
    w3 = _bits(np.array([[[0, 1]], [[1, 0]], [[0.5, 0.5]]], np.float32))
    w2 = _bits(np.array([[[1], [2]], [[-1], [0.5]], [[0.25], [-1]]], np.float32))
    r = O.moe_layer(x, wg, w1, w3, w2, 2)
    assert [sorted(map(int, row)) for row in r["ids"]] == [[0, 1], [0, 2]]
    assert list(map(int, r["ids"][1])) == [2, 0]
    a0, a1 = e / (e + 1), 1 / (e + 1)
    b0, b1 = e * e / (e * e + 1), 1 / (e * e + 1)
    np.testing.assert_allclose(r["weights"], [[a0, a1], [b0, b1]], rtol=1e-14, atol=0)
    h00, h01 = s(2.0), 2 * s(1.0)
    h12, h10 = -s(-2.0), -s(-1.0)
    out0 = [a0 * h00 - a1 * h01, a0 * 2 * h00 + a1 * 0.5 * h01]
    out1 = [b0 * 0.25 * h12 + b1 * h10, -b0 * h12 + b1 * 2 * h10]
    np.testing.assert_allclose(r["out"], [out0, out1], rtol=1e-13, atol=0)
    assert r["union_size"] == 3
    assert list(r["counts"]) == [2, 1, 1]
    assert list(r["offsets"]) == [0, 2, 3, 4]
    assert list(r["perm_token"]) == [0, 1, 0, 1]


# ---------------------------------------------------------------- gate

def _tie_logits(seed: int, T: int, E: int) -> np.ndarray:
    """Random logits on a coarse grid, so many exact ties occur."""
    rng = np.random.default_rng(seed)
    return rng.integers(-4, 5, size=(T, E)).astype(np.float64) * 0.25


def pin_selection_matches_stable_argsort(O) -> None:
    """Selection == numpy's stable argsort of the negated logits (ties keep the lower id)."""
    for seed, (T, E, k) in enumerate([(40, 16, 2), (30, 128, 8), (20, 9, 9), (25, 64, 4)]):
        logits = _tie_logits(seed, T, E)
        ref = np.argsort(-logits, axis=1, kind="stable")[:, :k]
        assert np.array_equal(O.select_experts(logits, k), ref)


def pin_weights_match_library_softmax(O) -> None:
    """Weights == scipy softmax over all E, gathered and renormalised; k = E is the plain softmax."""
    rng = np.random.default_rng(11)
    logits = rng.standard_normal((16, 32)) * 3
    for k in (1, 4, 32):
        ids = np.argsort(-logits, axis=1, kind="stable")[:, :k]
        w = O.routing_weights(logits, ids)
        p = softmax(logits, axis=1)
        sel = np.take_along_axis(p, ids, 1)
        np.testing.assert_allclose(w, sel / sel.sum(1, keepdims=True), rtol=1e-13, atol=1e-16)
        np.testing.assert_allclose(w.sum(1), 1.0, rtol=0, atol=1e-14)
        assert np.all(np.diff(w, axis=1) <= 0)  # follows the logit order
        if k == 1:
            assert np.all(w == 1.0)
    ids = np.argsort(-logits, axis=1, kind="stable")
    np.testing.assert_allclose(np.take_along_axis(softmax(logits, 1), ids, 1),
                               O.routing_weights(logits, ids), rtol=1e-13, atol=1e-16)


def pin_duplicate_gate_columns(O) -> None:
    """Experts with identical gate rows tie exactly; the lower id is selected first.

    Gate rows: e0 = 0, e1 = v, e2 = 0, e3 = -v, e4 = v, e5 = 2v and x = v, so the
    logits are (0, |v|^2, 0, -|v|^2, |v|^2, 2|v|^2): with k = 2 the picks are
    e5 then e1 (e4 ties with e1 and loses); with k = 3 they are e5, e1, e4.
    Then random gate rows where row 11 is a copy of row 4: whenever either is
    selected, 4 is selected, and 4 precedes 11.
    """
    v = np.array([0.5, -1.0, 0.25, 2.0], np.float32)
    wg = np.stack([0 * v, v, 0 * v, -v, v, 2 * v]).astype(np.float32)
    lg = O.gate_logits(v[None, :], wg)
    assert lg[0, 1] == lg[0, 4]
    assert list(map(int, O.select_experts(lg, 2)[0])) == [5, 1]
    assert list(map(int, O.select_experts(lg, 3)[0])) == [5, 1, 4]
    rng = np.random.default_rng(2)
    wg = rng.normal(0, 0.02, (16, 64)).astype(np.float32)
    wg[11] = wg[4]
    x = rng.standard_normal((200, 64)).astype(np.float32)
    lg = O.gate_logits(x, wg)
    ids = O.select_experts(lg, 2)
    assert np.array_equal(lg[:, 4], lg[:, 11])
    for row in ids:
        row = list(map(int, row))
        if 11 in row:
            assert 4 in row and row.index(4) < row.index(11)
    assert any(4 in row and 11 not in row for row in ids.tolist()), "no boundary tie exercised"


def pin_gate_logits_by_loops(O) -> None:
    """Gate logits equal an explicit double loop (no matmul) and torch's F.linear in float64."""
    s, x, wg, _, _, _ = _tiny_inputs(T=3)
    lg = O.gate_logits(x, wg)
    ref = torch.nn.functional.linear(torch.from_numpy(x).double(), torch.from_numpy(wg).double()).numpy()
    np.testing.assert_allclose(lg, ref, rtol=1e-13, atol=1e-15)
    for t in range(3):
        for e in (0, 7, 15):
            acc = math.fsum(float(x[t, h]) * float(wg[e, h]) for h in range(s.H))
            assert abs(lg[t, e] - acc) <= 1e-13


def pin_selection_gaps(O) -> None:
    """Gaps equal the difference of the k-th and (k+1)-th order statistics; inf when k == E."""
    logits = np.array([[3.0, 1.0, 2.0, 2.0], [0.0, 0.0, 0.0, 0.0]])
    np.testing.assert_array_equal(O.selection_gaps(logits, 1), [1.0, 0.0])
    np.testing.assert_array_equal(O.selection_gaps(logits, 2), [0.0, 0.0])
    np.testing.assert_array_equal(O.selection_gaps(logits, 3), [1.0, 0.0])
    assert np.all(np.isinf(O.selection_gaps(logits, 4)))


# ---------------------------------------------------------------- buckets

def _bucket_brute(ids: np.ndarray, E: int):
    pairs = sorted((int(e), t) for t in range(ids.shape[0]) for e in ids[t])
    return pairs


def pin_bucket_invariants(O) -> None:
    """Counts, offsets, slots and union against enumeration of (expert, token) pairs."""
    cases = []
    rng = np.random.default_rng(7)
    for T, E, K in [(8, 16, 2), (64, 128, 8), (33, 40, 5), (1, 4, 4), (17, 17, 1)]:
        cases.append((np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32), E))
    cases.append((np.tile(np.array([5, 2, 9], np.int32), (10, 1)), 12))  # identical tokens: U = k
    for ids, E in cases:
        T, K = ids.shape
        b = O.bucket(ids, E)
        pairs = _bucket_brute(ids, E)
        assert int(b["counts"].sum()) == T * K
        assert b["offsets"][0] == 0 and b["offsets"][E] == T * K
        assert np.all(np.diff(b["offsets"]) == b["counts"])
        # slot s holds the s-th pair in (expert, token) order
        slot_pairs = []
        for e in range(E):
            for s in range(b["offsets"][e], b["offsets"][e + 1]):
                slot_pairs.append((e, int(b["perm_token"][s])))
        assert slot_pairs == pairs
        for t in range(T):
            for j in range(K):
                s = int(b["pair_pos"][t, j])
                assert slot_pairs[s] == (int(ids[t, j]), t)
        assert list(b["union_ids"]) == sorted(set(int(e) for e in ids.ravel()))
        assert b["union_size"] == len(set(ids.ravel().tolist()))
        assert np.array_equal(b["counts"] > 0, np.isin(np.arange(E), b["union_ids"]))
    assert O.bucket(cases[-1][0], 12)["union_size"] == 3


ALL_PINS = [
    pin_dense_bruteforce_gate_routed,
    pin_dense_bruteforce_routed,
    pin_single_expert_is_dense_swiglu,
    pin_zero_input,
    pin_down_projection_linear,
    pin_closed_form_example,
    pin_selection_matches_stable_argsort,
    pin_weights_match_library_softmax,
    pin_duplicate_gate_columns,
    pin_gate_logits_by_loops,
    pin_selection_gaps,
    pin_bucket_invariants,
]
