"""CPU oracle for ELDR's expert signature, offline fit and online routing.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call this
module: only the tests and the benchmark's CPU-baseline leg use it.  It shares
no code with the native library and never imports it.

What it computes, in the paper's order and notation:

* Expert signature (Design, Expert Signature, construction steps).
  1. Count: c_r(l)[e], the request's prefill tokens routed to expert e at
     layer l (the block-summed counts of the signature cache).
  2. IDF reweight: w(l, e) = log((|C| + 1) / (df(l, e) + 1)), where df counts
     the calibration requests in which e fires at least once at l.
  3. Layer mask: keep the layers of S, stacked in the order of S.
  4. Normalise: s_r = x_r / ||x_r||_2.
* Signature quality rho (Design, Goal of Signature Design, the rho
  equation): the Spearman rank correlation, over given request pairs, between
  the cosine distance of their signatures and that of their decode-time
  activation probabilities p_i(l, e) (flattened and L2-normalised).
* Greedy layer selection (construction step 3): from an empty mask, append the
  layer whose inclusion gives the largest rho; the result is an ordering of
  all L layers, and N* is the prefix length where the cumulative rho peaks.
* Hungarian-balanced K-means (Design, Offline clustering): unit centroids;
  each centroid takes at most ceil(N/K) points; the assignment minimising the
  total cosine distance is found by the Hungarian algorithm (centroid k
  replicated ceil(N/K) times as columns of the cost matrix); a centroid is
  the normalised mean of its points; iterate until the assignment repeats.
* Locality-band routing (Design, Online routing): s* = max_k cos(s, c_k);
  among the workers with cos(s, c_k) >= s* - tau pick the one with the fewest
  in-flight requests.

Readings where the paper is silent (listed in the design notes): ties in
greedy selection go to the lower layer index and N* to the shorter prefix;
K-means starts from given initial points (the caller draws them) and stops
after max_iters if the assignment keeps changing; a centroid with no points
keeps its previous value; a zero count vector gives a zero signature;
routing ties in load go to the higher similarity, then the lower worker index.

Arithmetic is float64 throughout.
"""
from __future__ import annotations

import numpy as np
from scipy.optimize import linear_sum_assignment
from scipy.stats import spearmanr


def idf_table(counts: np.ndarray) -> np.ndarray:
    """w(l, e) = log((|C| + 1) / (df(l, e) + 1)) from calibration counts [N, L, E]."""
    counts = np.asarray(counts)
    n = counts.shape[0]
    df = (counts > 0).sum(axis=0)
    return np.log((n + 1.0) / (df + 1.0))


def signature(counts: np.ndarray, idf: np.ndarray, layers) -> np.ndarray:
    """s = x / ||x||_2 with x the IDF-weighted counts of the kept layers, stacked in order."""
    counts = np.asarray(counts, dtype=np.float64)
    x = np.concatenate([counts[l] * idf[l] for l in layers]) if len(layers) else np.zeros(0)
    n = np.sqrt(np.sum(x * x))
    return x / n if n > 0 else np.zeros_like(x)


def cos_dist(a: np.ndarray, b: np.ndarray) -> float:
    """1 - cosine similarity; 1 when either vector is zero."""
    na = np.sqrt(np.sum(a * a))
    nb = np.sqrt(np.sum(b * b))
    if na == 0 or nb == 0:
        return 1.0
    return 1.0 - float(np.dot(a, b) / (na * nb))


def rho(S: np.ndarray, P: np.ndarray, pairs: np.ndarray) -> float:
    """Spearman correlation between pairwise cosine distances of S rows and of P rows."""
    ds = [cos_dist(S[i], S[j]) for i, j in pairs]
    dp = [cos_dist(P[i], P[j]) for i, j in pairs]
    if np.ptp(ds) == 0 or np.ptp(dp) == 0:
        return 0.0
    return float(spearmanr(ds, dp).statistic)


def greedy_layers(counts: np.ndarray, idf: np.ndarray, P: np.ndarray, pairs: np.ndarray
                  ) -> tuple[list[int], list[float], int]:
    """Greedy layer ordering by rho; returns (order, cumulative rho per prefix, N*)."""
    counts = np.asarray(counts)
    L = counts.shape[1]
    chosen: list[int] = []
    curve: list[float] = []
    remaining = list(range(L))
    while remaining:
        best, best_rho = None, -np.inf
        for l in remaining:  # ascending, so ties keep the lower layer
            trial = chosen + [l]
            S = np.stack([signature(counts[i], idf, trial) for i in range(counts.shape[0])])
            r = rho(S, P, pairs)
            if r > best_rho:
                best, best_rho = l, r
        chosen.append(best)
        remaining.remove(best)
        curve.append(best_rho)
    n_star = int(np.argmax(curve)) + 1  # first peak: the shorter prefix on ties
    return chosen, curve, n_star


def balanced_kmeans(S: np.ndarray, K: int, init: np.ndarray, max_iters: int = 50
                    ) -> tuple[np.ndarray, np.ndarray, int]:
    """Hungarian-balanced K-means on unit rows of S [N, d] from initial points `init` [K].

    Returns (centroids [K, d], assignment [N], iterations run).
    """
    S = np.asarray(S, dtype=np.float64)
    N = S.shape[0]
    cap = -(-N // K)
    C = S[np.asarray(init)].copy()
    C /= np.linalg.norm(C, axis=1, keepdims=True)
    assign = None
    it = 0
    for it in range(1, max_iters + 1):
        cost = 1.0 - S @ C.T                       # cosine distance (rows and centroids are unit)
        rows, cols = linear_sum_assignment(np.repeat(cost, cap, axis=1))
        new = np.empty(N, dtype=np.int64)
        new[rows] = cols // cap
        for k in range(K):
            pts = S[new == k]
            if len(pts):
                m = pts.mean(axis=0)
                nm = np.linalg.norm(m)
                if nm > 0:
                    C[k] = m / nm
        if assign is not None and np.array_equal(new, assign):
            assign = new
            break
        assign = new
    return C, assign, it


def route(s: np.ndarray, centroids: np.ndarray, loads: np.ndarray, tau: float) -> int:
    """Locality-band routing: fewest in-flight requests among workers with sim >= s* - tau."""
    sims = np.array([1.0 - cos_dist(s, c) for c in centroids])
    top = sims.max()
    band = [k for k in range(len(centroids)) if sims[k] >= top - tau]
    return min(band, key=lambda k: (int(loads[k]), -sims[k], k))
