"""The routing oracle against its pins, and the pins against planted mistakes.

Pins: closed forms (IDF, the no-ties Spearman formula, unit signatures),
brute force (every balanced partition of a tiny set; the best single layer),
recovery of well-separated equal clusters, the capacity bound on skewed data,
and the two limits of locality-band routing (tau = 0: nearest centroid;
tau = 1 with non-negative signatures: fewest in-flight requests).
"""
import importlib.util
import itertools
import os

import numpy as np
import pytest

from oracle import routing as RO

SRC = os.path.join(os.path.dirname(RO.__file__), "routing.py")


def unit_rows(X):
    return X / np.linalg.norm(X, axis=1, keepdims=True)


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def pin_idf_closed_form(O):
    counts = np.zeros((4, 1, 3), np.int64)  # 4 requests, 1 layer, 3 experts
    counts[:, 0, 0] = [1, 2, 0, 5]           # fires in 3 requests
    counts[:, 0, 1] = [1, 1, 1, 1]           # fires in all 4
    w = O.idf_table(counts)                  # expert 2 never fires
    assert np.allclose(w[0], [np.log(5 / 4), np.log(5 / 5), np.log(5 / 1)], rtol=0, atol=1e-15)


def pin_signature_unit_and_order(O):
    rng = np.random.default_rng(1)
    counts = rng.integers(0, 9, (4, 6)).astype(np.int64)
    idf = np.ones((4, 6))
    s = O.signature(counts, idf, [0, 1, 2, 3])
    x = counts.reshape(-1).astype(np.float64)
    assert np.allclose(s, x / np.sqrt((x * x).sum()), atol=1e-15)
    idf = rng.random((4, 6))
    s2 = O.signature(counts, idf, [2, 0])
    x2 = np.concatenate([counts[2] * idf[2], counts[0] * idf[0]])
    assert np.allclose(s2, x2 / np.linalg.norm(x2), atol=1e-15)
    assert abs(np.linalg.norm(s2) - 1) < 1e-12
    assert not O.signature(np.zeros((2, 3)), np.ones((2, 3)), [0, 1]).any()


def pin_rho_no_ties_formula(O):
    rng = np.random.default_rng(2)
    S = unit_rows(rng.random((12, 5)))
    P = unit_rows(rng.random((12, 7)))
    pairs = np.array(list(itertools.combinations(range(12), 2))[:40])
    ds = np.array([1 - S[i] @ S[j] for i, j in pairs])
    dp = np.array([1 - P[i] @ P[j] for i, j in pairs])
    rs = np.argsort(np.argsort(ds))
    rp = np.argsort(np.argsort(dp))
    n = len(pairs)
    ref = 1 - 6 * np.sum((rs - rp) ** 2) / (n * (n * n - 1))
    assert abs(O.rho(S, P, pairs) - ref) < 1e-12
    assert abs(O.rho(S, S, pairs) - 1) < 1e-12


def pin_greedy_first_layer_is_best_single(O):
    rng = np.random.default_rng(3)
    N, L, E = 30, 4, 8
    counts = rng.integers(0, 5, (N, L, E))
    P = unit_rows(counts[:, 1].astype(float) + 0.3 * rng.random((N, E)))  # layer 1 predicts P
    idf = O.idf_table(counts)
    pairs = np.array(list(itertools.combinations(range(N), 2)))
    order, curve, n_star = O.greedy_layers(counts, idf, P, pairs)
    singles = [O.rho(np.stack([O.signature(counts[i], idf, [l]) for i in range(N)]), P, pairs)
               for l in range(L)]
    assert order[0] == int(np.argmax(singles)) == 1
    assert abs(curve[0] - max(singles)) < 1e-12
    assert sorted(order) == list(range(L))
    assert n_star == int(np.argmax(curve)) + 1 and 1 <= n_star <= L


def pin_kmeans_brute_force_assignment(O):
    rng = np.random.default_rng(4)
    S = unit_rows(rng.random((6, 3)))
    C, assign, _ = O.balanced_kmeans(S, 2, init=np.array([0, 5]), max_iters=1)
    # one iteration: the assignment is optimal for the initial centroids
    C0 = S[[0, 5]]
    best = min(sum(1 - S[i] @ C0[0 if i in part else 1] for i in range(6))
               for part in itertools.combinations(range(6), 3))
    got = sum(1 - S[i] @ C0[assign[i]] for i in range(6))
    assert abs(got - best) < 1e-12
    assert np.bincount(assign, minlength=2).max() <= 3


def pin_kmeans_recovers_separated_clusters(O):
    rng = np.random.default_rng(5)
    centers = np.eye(4)
    S = unit_rows(np.repeat(centers, 25, axis=0) + 0.05 * rng.random((100, 4)))
    C, assign, _ = O.balanced_kmeans(S, 4, init=np.array([0, 30, 60, 90]))
    for k in range(4):
        assert len(set(assign[25 * k:25 * k + 25])) == 1
    assert len(set(assign)) == 4
    assert np.allclose(np.linalg.norm(C, axis=1), 1)


def pin_kmeans_capacity_on_skewed_data(O):
    rng = np.random.default_rng(6)
    dense = unit_rows(np.array([1.0, 0, 0]) + 0.05 * rng.random((70, 3)))
    sparse = unit_rows(rng.random((30, 3)))
    S = np.vstack([dense, sparse])
    C, assign, _ = O.balanced_kmeans(S, 4, init=np.array([0, 1, 2, 3]))
    assert np.bincount(assign, minlength=4).max() <= 25
    assert len(set(assign)) == 4


def pin_route_limits(O):
    rng = np.random.default_rng(7)
    C = unit_rows(rng.random((6, 5)))
    s = unit_rows(rng.random((1, 5)))[0]
    sims = C @ s
    loads = np.array([5, 1, 4, 0, 2, 3])
    assert O.route(s, C, loads, 0.0) == int(np.argmax(sims))
    assert O.route(s, C, loads, 1.0) == 3  # non-negative vectors: every worker is in the band
    # a band of the two most similar workers picks the less loaded one
    order = np.argsort(-sims)
    tau = (sims[order[0]] - sims[order[1]]) + 1e-9
    if sims[order[1]] - sims[order[2]] > 1e-6:
        expect = min(order[:2], key=lambda k: loads[k])
        assert O.route(s, C, loads, tau) == expect


ALL_PINS = [pin_idf_closed_form, pin_signature_unit_and_order, pin_rho_no_ties_formula,
            pin_greedy_first_layer_is_best_single, pin_kmeans_brute_force_assignment,
            pin_kmeans_recovers_separated_clusters, pin_kmeans_capacity_on_skewed_data,
            pin_route_limits]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(RO)


# ---------------------------------------------------------------------------
# planted mistakes
# ---------------------------------------------------------------------------

def _mutant(old: str, new: str):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    spec = importlib.util.spec_from_loader("routing_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src.replace(old, new), "routing_mutant", "exec"), mod.__dict__)
    return mod


MUTATIONS = {
    "idf_no_plus_one": ("return np.log((n + 1.0) / (df + 1.0))", "return np.log(n / (df + 1.0))"),
    "idf_inverted": ("return np.log((n + 1.0) / (df + 1.0))", "return np.log((df + 1.0) / (n + 1.0))"),
    "no_normalise": ("return x / n if n > 0 else np.zeros_like(x)", "return x"),
    "idf_not_applied": ("x = np.concatenate([counts[l] * idf[l] for l in layers])",
                        "x = np.concatenate([counts[l] for l in layers])"),
    "rho_pearson": ("return float(spearmanr(ds, dp).statistic)", "return float(np.corrcoef(ds, dp)[0, 1])"),
    "greedy_worst_layer": ("if r > best_rho:", "if -r > best_rho:"),
    "n_star_last": ("n_star = int(np.argmax(curve)) + 1", "n_star = len(curve)"),
    "kmeans_no_capacity": ("rows, cols = linear_sum_assignment(np.repeat(cost, cap, axis=1))",
                           "rows, cols = np.arange(N), np.argmin(cost, axis=1) * cap"),
    "kmeans_max_distance": ("cost = 1.0 - S @ C.T", "cost = S @ C.T"),
    "route_ignores_load": ("return min(band, key=lambda k: (int(loads[k]), -sims[k], k))",
                           "return min(band, key=lambda k: (-sims[k], k))"),
    "route_ignores_band": ("band = [k for k in range(len(centroids)) if sims[k] >= top - tau]",
                           "band = list(range(len(centroids)))"),
}


def _caught(mod) -> bool:
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception:
            return True
    return False


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    old, new = MUTATIONS[name]
    assert _caught(_mutant(old, new)), f"no pin catches mutation {name}"
