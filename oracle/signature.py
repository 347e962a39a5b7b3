"""CPU oracle for ELDR's block-granular expert-signature cache (NumPy, integers).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call this
module: only the tests and the benchmark's CPU-baseline leg use it.  It shares
no code with the HIP library and never imports it.

What it computes (Design, Prefix Cache Coherence):

* The signature cache holds one row per KV-cache block, indexed by the block
  id, with one small integer per (MoE layer, expert).
* When prefill writes a token's K/V into a block, the top-k experts the gate
  picked for that token at every MoE layer are added to that block's row.
* A reused block starts from a zero row (the cache follows the KV cache's
  block lifecycle).
* A request's signature counts are the sum of the rows of the blocks its KV
  cache spans.  This is exact under prefix-cache hits, because each cached
  block still holds the picks of the tokens it stores.
* The raw quantity this equals is the per-layer count of prompt tokens routed
  to each expert (Design, Expert Signature, the counting step).

Readings where the paper is silent (listed in the design notes):

* a token whose block id is negative has no KV slot and is not recorded;
* ids outside [0, E) or block ids outside the cache are skipped and counted
  as rejected picks;
* cells are int8 in the cache, so a block holds at most 127 tokens in its
  lifetime; per-request sums are int32, exact at any prompt length.

All arithmetic here is exact integer counting in int64.

Pins: checked in the CPU suite against np.bincount / np.add.at, an explicit
dict count on tiny inputs, and the prefix-cache scenarios the paper names
(cold prefill, partial hit, full hit, chunked prefill, eviction and reuse).
"""
from __future__ import annotations

import numpy as np


def new_cache(num_blocks: int, L: int, E: int) -> np.ndarray:
    """An empty signature cache, int64 [num_blocks, L, E]: one row per KV block."""
    return np.zeros((num_blocks, L, E), dtype=np.int64)


def capture(sig: np.ndarray, ids: np.ndarray, token_block: np.ndarray,
            layer0: int = 0) -> tuple[np.ndarray, int]:
    """Add one forward's picks to the cache (Design, Prefix Cache Coherence).

    ids [n_layers, T, K]: the experts the gate picked for each new token at MoE
    layers layer0 .. layer0 + n_layers - 1.  token_block [T]: the KV block each
    new token is written to (negative: not recorded).  For every layer l,
    token t and pick j: sig[token_block[t], layer0 + l, ids[l, t, j]] += 1.
    Returns the updated cache (a copy) and the number of rejected picks.
    """
    out = np.array(sig, dtype=np.int64, copy=True)
    nb, L, E = out.shape
    ids = np.asarray(ids)
    n_layers, T, K = ids.shape
    rejected = 0
    for l in range(n_layers):
        for t in range(T):
            b = int(token_block[t])
            if b < 0:
                continue
            for j in range(K):
                e = int(ids[l, t, j])
                if b >= nb or not (0 <= e < E) or not (0 <= layer0 + l < L):
                    rejected += 1
                    continue
                out[b, layer0 + l, e] += 1
    return out, rejected


def reset(sig: np.ndarray, blocks) -> np.ndarray:
    """Zero the rows of blocks handed to a new request (the KV block lifecycle)."""
    out = np.array(sig, dtype=np.int64, copy=True)
    for b in blocks:
        if 0 <= int(b) < out.shape[0]:
            out[int(b)] = 0
    return out


def request_counts(sig: np.ndarray, blocks) -> np.ndarray:
    """A request's counts s_r = sum over its blocks b of sig[b], int64 [L, E]."""
    out = np.zeros(sig.shape[1:], dtype=np.int64)
    for b in blocks:
        out += sig[int(b)]
    return out


def prompt_counts(ids: np.ndarray, E: int) -> np.ndarray:
    """Per-layer count of a prompt's tokens routed to each expert, int64 [L, E].

    ids [L, T, K] are the picks of every prompt token at every MoE layer (the
    counting step of the signature: c_r(l)[e] = tokens routed to e at layer l).
    """
    ids = np.asarray(ids)
    L = ids.shape[0]
    out = np.zeros((L, E), dtype=np.int64)
    for l in range(L):
        for e in ids[l].reshape(-1):
            out[l, int(e)] += 1
    return out
