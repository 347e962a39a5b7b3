/*
 * eldr_route.h -- ELDR's expert signature, offline fit and online routing
 * (arXiv 2607.00466, Design: Expert Signature, Offline clustering, Online
 * routing), as a native host library (no GPU work; the counts come from the
 * signature cache, eldr_signature.h).
 *
 * Plain host pointers and sizes; the caller owns every buffer; no call keeps
 * state.  Every call returns MOE_OK (0) or a negative MOE_ERR_* code
 * (eldr_moe.h); MOE_ERR_INVALID for null pointers, non-positive sizes or
 * indices out of range.  Layouts are row-major.  Arithmetic is double inside;
 * float arrays are widened exactly.
 */
#ifndef ELDR_ROUTE_H_
#define ELDR_ROUTE_H_

#include <stddef.h>
#include <stdint.h>

#include "eldr_moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * eldr_idf -- IDF table of the signature (construction step 2):
 *   idf[l, e] = log((N + 1) / (df(l, e) + 1)),
 * df(l, e) = number of the N calibration requests whose count at (l, e) is
 * positive.  counts [N, L, E] int32 (prefill counts per request), idf [L, E].
 */
int eldr_idf(const int32_t* counts, int32_t N, int32_t L, int32_t E, float* idf);

/*
 * eldr_signature -- one request's signature (construction steps 1-4): the
 * counts [L, E] of the kept layers `layers` [n_layers] (in that order), each
 * row multiplied by its IDF row, stacked, divided by the L2 norm (all zeros
 * when the stacked vector is zero).  s [n_layers * E].
 */
int eldr_signature(const int32_t* counts, const float* idf, int32_t L, int32_t E,
                   const int32_t* layers, int32_t n_layers, float* s);

/*
 * eldr_rho -- signature quality (the rho equation): the Spearman rank
 * correlation (average ranks on ties) between cos-dist(S[i], S[j]) and
 * cos-dist(P[i], P[j]) over the n_pairs pairs `pairs` [n_pairs, 2].
 * cos-dist(a, b) = 1 - a.b / (|a| |b|), and 1 when a or b is zero.  S [N, d]
 * signatures, P [N, dp] decode-time activation probabilities.  *rho is 0 when
 * either list of distances is constant.
 */
int eldr_rho(const float* S, int32_t N, int32_t d, const float* P, int32_t dp,
             const int32_t* pairs, int32_t n_pairs, double* rho);

/*
 * eldr_greedy_layers -- the layer mask (construction step 3): from an empty
 * mask, repeatedly append the layer whose inclusion gives the largest rho
 * (ties to the lower layer index) until every layer is ordered.  order [L]
 * receives the ordering, curve [L] the rho of each prefix, *n_star the prefix
 * length with the largest rho (the shortest on ties).  counts [N, L, E],
 * idf [L, E], P [N, dp], pairs [n_pairs, 2].
 */
int eldr_greedy_layers(const int32_t* counts, int32_t N, int32_t L, int32_t E, const float* idf,
                       const float* P, int32_t dp, const int32_t* pairs, int32_t n_pairs,
                       int32_t* order, double* curve, int32_t* n_star);

/*
 * eldr_balanced_kmeans -- Hungarian-balanced K-means (Design, Offline
 * clustering) on the unit rows of S [N, d]: each of the K unit centroids
 * takes at most ceil(N / K) points, and the assignment that minimises the
 * total cosine distance is solved exactly (Hungarian algorithm on the N x
 * K*ceil(N/K) matrix of centroid copies); each centroid then becomes the
 * normalised mean of its points (a centroid with no points keeps its value).
 * Starts from the points init [K] (drawn by the caller) and stops when the
 * assignment repeats or after max_iters iterations.  centroids [K, d],
 * assign [N], *iters = iterations run.
 */
int eldr_balanced_kmeans(const float* S, int32_t N, int32_t d, int32_t K, const int32_t* init,
                         int32_t max_iters, float* centroids, int32_t* assign, int32_t* iters);

/*
 * eldr_route -- locality-band routing (Design, Online routing): with
 * s_k = cos(s, centroids[k]) and s* = max_k s_k, among the workers with
 * s_k >= s* - tau pick the one with the fewest in-flight requests loads[k];
 * ties go to the higher s_k, then the lower k.  s [d], centroids [K, d],
 * loads [K].  *worker receives the choice.  tau must be finite and >= 0
 * (the paper sweeps it over [0, 1]), else MOE_ERR_INVALID.  A non-finite
 * signature or centroid leaves no worker in the band: *worker = -1 and
 * MOE_ERR_INVALID.
 */
int eldr_route(const float* s, int32_t d, const float* centroids, int32_t K,
               const int32_t* loads, float tau, int32_t* worker);

/*
 * eldr_route_batch -- route R requests in order with eldr_route, each choice
 * adding one in-flight request to its worker: S [R, d], loads [K] (in/out),
 * workers [R].  Errors as eldr_route; routing stops at the first request with
 * no worker, which and every later one get workers[r] = -1 and add no load
 * (the requests before it stay routed).
 */
int eldr_route_batch(const float* S, int32_t R, int32_t d, const float* centroids, int32_t K,
                     int32_t* loads, float tau, int32_t* workers);

#ifdef __cplusplus
}
#endif

#endif  /* ELDR_ROUTE_H_ */
