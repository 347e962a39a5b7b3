"""The signature-cache oracle against its pins, and the pins against planted mistakes.

Pins: library routines (np.add.at, np.bincount), an explicit dict count on
tiny inputs, and the prefix-cache scenarios of Design, Prefix Cache Coherence
(cold prefill, partial hit, full hit, chunked prefill, eviction and reuse),
where the block-summed counts must equal the prompt's own per-layer counts.
"""
import importlib.util
import os
from collections import Counter

import numpy as np
import pytest

from oracle import signature as sig_oracle
from paper_2607_00466_amd import synth

SRC = os.path.join(os.path.dirname(sig_oracle.__file__), "signature.py")
B = 16  # KV block size (tokens) used by the scenarios


def blocks_for(positions, table):
    """Block of each token position, from a request's block table."""
    return np.array([table[p // B] for p in positions], dtype=np.int64)


def bincount_counts(ids, E):
    """Per-layer expert counts through np.bincount (the library pin)."""
    return np.stack([np.bincount(ids[l].reshape(-1), minlength=E) for l in range(ids.shape[0])])


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def pin_capture_matches_add_at(O):
    L, T, K, E, NB = 3, 100, 4, 32, 12
    ids = synth.prefill_picks(L, T, E, K, seed=3)
    rng = np.random.default_rng(5)
    tb = rng.integers(0, NB, T)
    got, rej = O.capture(O.new_cache(NB, L, E), ids, tb)
    ref = np.zeros((NB, L, E), np.int64)
    for l in range(L):
        np.add.at(ref, (np.repeat(tb, K), l, ids[l].reshape(-1)), 1)
    assert rej == 0
    assert np.array_equal(got, ref)


def pin_capture_dict_count(O):
    ids = np.array([[[0, 2], [1, 2], [2, 0]], [[3, 1], [3, 0], [1, 2]]])  # [L=2, T=3, K=2]
    tb = np.array([1, 1, 0])
    got, _ = O.capture(O.new_cache(2, 2, 4), ids, tb)
    c = Counter()
    for l in range(2):
        for t in range(3):
            for j in range(2):
                c[(int(tb[t]), l, int(ids[l, t, j]))] += 1
    ref = np.zeros((2, 2, 4), np.int64)
    for (b, l, e), n in c.items():
        ref[b, l, e] = n
    assert np.array_equal(got, ref)
    assert got[1, 0, 2] == 2 and got[0, 1, 2] == 1


def pin_prompt_counts_bincount(O):
    ids = synth.prefill_picks(4, 57, 64, 8, seed=7, skew=1.1)
    assert np.array_equal(O.prompt_counts(ids, 64), bincount_counts(ids, 64))


def pin_cold_prefill(O):
    L, E, K, T = 4, 32, 4, 70  # 70 tokens: 4 full blocks and a partial one
    ids = synth.prefill_picks(L, T, E, K, seed=8)
    table = [9, 2, 7, 0, 5]
    sig, _ = O.capture(O.new_cache(10, L, E), ids, blocks_for(range(T), table))
    assert np.array_equal(O.request_counts(sig, table), bincount_counts(ids, E))


def pin_partial_hit(O):
    # Request A prefills 80 tokens; request B shares A's first 48 tokens (three
    # full cached blocks) and prefills its 40 new tokens into fresh blocks.
    L, E, K = 3, 32, 4
    a_ids = synth.prefill_picks(L, 80, E, K, seed=9)
    a_table = [0, 1, 2, 3, 4]
    sig, _ = O.capture(O.new_cache(12, L, E), a_ids, blocks_for(range(80), a_table))
    new_ids = synth.prefill_picks(L, 40, E, K, seed=10)
    b_ids = np.concatenate([a_ids[:, :48], new_ids], axis=1)
    b_table = [0, 1, 2, 8, 6, 11]
    sig, _ = O.capture(sig, new_ids, blocks_for(range(48, 88), b_table))
    assert np.array_equal(O.request_counts(sig, b_table), bincount_counts(b_ids, E))
    # A's own counts are untouched by B's prefill
    assert np.array_equal(O.request_counts(sig, a_table), bincount_counts(a_ids, E))


def pin_full_hit(O):
    L, E, K = 2, 16, 2
    ids = synth.prefill_picks(L, 32, E, K, seed=11)
    table = [3, 1]
    sig, _ = O.capture(O.new_cache(4, L, E), ids, blocks_for(range(32), table))
    # a second request with the same prompt prefills nothing and reads the same blocks
    assert np.array_equal(O.request_counts(sig, table), bincount_counts(ids, E))


def pin_chunked_prefill(O):
    L, E, K, T = 3, 32, 4, 60
    ids = synth.prefill_picks(L, T, E, K, seed=12)
    table = [4, 0, 2, 1]
    tb = blocks_for(range(T), table)
    one, _ = O.capture(O.new_cache(5, L, E), ids, tb)
    cut = 23  # mid-block: block 0 of the table is filled by both forwards
    two, _ = O.capture(O.new_cache(5, L, E), ids[:, :cut], tb[:cut])
    two, _ = O.capture(two, ids[:, cut:], tb[cut:])
    assert np.array_equal(one, two)


def pin_eviction_and_reuse(O):
    L, E, K = 2, 16, 2
    old = synth.prefill_picks(L, 16, E, K, seed=13)
    sig, _ = O.capture(O.new_cache(3, L, E), old, np.full(16, 1))
    new = synth.prefill_picks(L, 10, E, K, seed=14)
    sig = O.reset(sig, [1])
    sig, _ = O.capture(sig, new, np.full(10, 1))
    assert np.array_equal(sig[1], bincount_counts(new, E))
    assert not sig[0].any() and not sig[2].any()


def pin_order_invariance(O):
    L, E, K, T = 2, 32, 4, 50
    ids = synth.prefill_picks(L, T, E, K, seed=15)
    tb = np.random.default_rng(16).integers(0, 6, T)
    p = np.random.default_rng(17).permutation(T)
    a, _ = O.capture(O.new_cache(6, L, E), ids, tb)
    b, _ = O.capture(O.new_cache(6, L, E), ids[:, p], tb[p])
    assert np.array_equal(a, b)


def pin_layer_offset(O):
    # one layer at a time with layer0 equals all layers at once
    L, E, K, T = 4, 16, 2, 20
    ids = synth.prefill_picks(L, T, E, K, seed=18)
    tb = np.arange(T) // B
    whole, _ = O.capture(O.new_cache(2, L, E), ids, tb)
    part = O.new_cache(2, L, E)
    for l in range(L):
        part, _ = O.capture(part, ids[l:l + 1], tb, layer0=l)
    assert np.array_equal(whole, part)


def pin_rejections(O):
    ids = np.array([[[0, 5], [1, -1], [2, 3]]])  # E = 4: ids 5 and -1 are invalid
    tb = np.array([0, 7, -1])  # block 7 is outside a 2-block cache; -1 is not recorded
    sig, rej = O.capture(O.new_cache(2, 1, 4), ids, tb)
    assert rej == 3  # id 5, and both picks of the token in block 7
    assert sig[0, 0].tolist() == [1, 0, 0, 0] and not sig[1].any()


ALL_PINS = [pin_capture_matches_add_at, pin_capture_dict_count, pin_prompt_counts_bincount,
            pin_cold_prefill, pin_partial_hit, pin_full_hit, pin_chunked_prefill,
            pin_eviction_and_reuse, pin_order_invariance, pin_layer_offset, pin_rejections]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(sig_oracle)


# ---------------------------------------------------------------------------
# planted mistakes: each must fail at least one pin
# ---------------------------------------------------------------------------

def _mutant(old: str, new: str):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    spec = importlib.util.spec_from_loader("signature_mutant", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src.replace(old, new), "signature_mutant", "exec"), mod.__dict__)
    return mod


MUTATIONS = {
    "next_block": ("out[b, layer0 + l, e] += 1", "out[min(b + 1, nb - 1), layer0 + l, e] += 1"),
    "layer_ignored": ("out[b, layer0 + l, e] += 1", "out[b, layer0, e] += 1"),
    "top1_only": ("for j in range(K):", "for j in range(1):"),
    "negative_block_recorded": ("if b < 0:\n                continue", "if b < -1:\n                continue"),
    "reset_is_noop": ("out[int(b)] = 0", "out[int(b)] = out[int(b)]"),
    "request_first_block_only": ("out += sig[int(b)]", "out += sig[int(blocks[0])]"),
    "prompt_counts_layer0": ("for e in ids[l].reshape(-1):", "for e in ids[0].reshape(-1):"),
    "rejects_not_counted": ("rejected += 1", "rejected += 0"),
    "double_count": ("out[b, layer0 + l, e] += 1", "out[b, layer0 + l, e] += 1 + (e == 0)"),
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
