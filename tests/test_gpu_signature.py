"""GPU parity of the expert-signature cache calls against the CPU oracle.

Integer work: every comparison is bit-exact.  Scenarios follow Design, Prefix
Cache Coherence (cold prefill, partial and full prefix hits, chunked prefill,
eviction and reuse); the sizes span several workgroups and ragged tails, and
one case uses the 48-layer, 128-expert, top-8 shape with a 2048-token
prefill.
"""
import numpy as np
import pytest
import torch

from oracle import signature as SO
from paper_2607_00466_amd import binding as B
from paper_2607_00466_amd import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

BS = 16  # KV block size used by the scenarios


def dev(a, dtype=torch.int32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).cuda()


class Cache:
    """A device cache and the oracle's copy of it, driven through the same calls."""

    def __init__(self, num_blocks, L, E):
        self.L, self.E = L, E
        self.sig = torch.zeros((num_blocks, L, E), dtype=torch.int8, device="cuda")
        self.ref = SO.new_cache(num_blocks, L, E)
        self.rejected = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.ref_rejected = 0

    def capture(self, ids, token_block, layer0=0):
        B.moe_sig_capture(dev(ids), dev(token_block), layer0, self.L, self.E, self.sig, self.rejected)
        self.ref, r = SO.capture(self.ref, ids, token_block, layer0)
        self.ref_rejected += r

    def reset(self, blocks):
        B.moe_sig_reset(dev(blocks), self.sig)
        self.ref = SO.reset(self.ref, blocks)

    def check(self, label):
        torch.cuda.synchronize()
        got = self.sig.cpu().numpy().astype(np.int64)
        assert np.array_equal(got, self.ref), label
        assert int(self.rejected.item()) == self.ref_rejected, label

    def request_counts(self, tables):
        R = len(tables)
        mb = max(1, max(len(t) for t in tables))
        table = np.full((R, mb), -1, np.int32)
        for r, t in enumerate(tables):
            table[r, :len(t)] = t
        n = np.array([len(t) for t in tables], np.int32)
        out = B.moe_sig_request_counts(self.sig, dev(table), dev(n))
        torch.cuda.synchronize()
        return out.cpu().numpy().astype(np.int64)


def blocks_for(positions, table):
    return np.array([table[p // BS] for p in positions], np.int32)


def test_capture_random_blocks_bit_exact():
    G.say("case: signature capture, L=5 E=64 K=8 T=1000 (ragged) into 70 random blocks")
    L, E, K, T = 5, 64, 8, 1000
    c = Cache(70, L, E)
    ids = synth.prefill_picks(L, T, E, K, seed=1, skew=1.1)
    tb = np.random.default_rng(2).integers(0, 70, T).astype(np.int32)
    c.capture(ids, tb)
    c.check("random capture")


def test_full_shape_prefill_and_request_counts():
    G.say("case: signature capture, 48 layers, E=128, top-8, 2048-token prefill, 16-token blocks")
    L, E, K, T = 48, 128, 8, 2048
    c = Cache(256, L, E)
    ids = synth.prefill_picks(L, T, E, K, seed=3, skew=1.1)
    table = list(np.random.default_rng(4).permutation(256)[:T // BS])
    c.capture(ids, blocks_for(range(T), table))
    c.check("2048-token prefill")
    got = c.request_counts([table])
    assert np.array_equal(got[0], SO.prompt_counts(ids, E))


def test_prefix_cache_scenarios():
    G.say("case: signature cache scenarios: cold, partial hit, full hit, chunked, eviction")
    L, E, K = 6, 32, 4
    c = Cache(40, L, E)
    # cold prefill of A (80 tokens, blocks 0..4)
    a_ids = synth.prefill_picks(L, 80, E, K, seed=5)
    a_table = [0, 1, 2, 3, 4]
    c.capture(a_ids, blocks_for(range(80), a_table))
    c.check("cold")
    # B shares A's first 48 tokens (3 cached blocks) and prefills 40 new tokens in two chunks
    new = synth.prefill_picks(L, 40, E, K, seed=6)
    b_table = [0, 1, 2, 9, 17, 33]
    tb = blocks_for(range(48, 88), b_table)
    c.capture(new[:, :13], tb[:13])
    c.capture(new[:, 13:], tb[13:])
    c.check("partial hit, chunked")
    b_ids = np.concatenate([a_ids[:, :48], new], axis=1)
    # C is a full hit on A: nothing to prefill
    got = c.request_counts([a_table, b_table, a_table])
    assert np.array_equal(got[0], SO.prompt_counts(a_ids, E))
    assert np.array_equal(got[1], SO.prompt_counts(b_ids, E))
    assert np.array_equal(got[2], got[0])
    # A's last block is evicted and reused by D
    c.reset([4])
    d_ids = synth.prefill_picks(L, 9, E, K, seed=7)
    c.capture(d_ids, np.full(9, 4, np.int32))
    c.check("eviction and reuse")
    assert np.array_equal(c.request_counts([[4]])[0], SO.prompt_counts(d_ids, E))


def test_layer_by_layer_equals_one_pass():
    G.say("case: signature capture one layer at a time (layer0) vs all layers at once")
    L, E, K, T = 7, 64, 8, 300
    ids = synth.prefill_picks(L, T, E, K, seed=8)
    tb = (np.arange(T) // BS).astype(np.int32)
    a = Cache(20, L, E)
    a.capture(ids, tb)
    b = Cache(20, L, E)
    for l in range(L):
        b.capture(ids[l:l + 1], tb, layer0=l)
    a.check("one pass")
    b.check("per layer")
    assert torch.equal(a.sig, b.sig)


def test_rejections_and_unrecorded_tokens():
    G.say("case: signature capture with bad ids, out-of-cache blocks and unrecorded tokens")
    L, E, K, T = 2, 16, 4, 50
    ids = synth.prefill_picks(L, T, E, K, seed=9)
    ids[0, 3, 1] = E + 5
    ids[1, 7, 0] = -2
    tb = (np.arange(T) % 6).astype(np.int32)
    tb[10] = 6      # outside a 6-block cache
    tb[11] = -1     # not recorded
    c = Cache(6, L, E)
    c.capture(ids, tb)
    c.check("rejections")
    assert c.ref_rejected == 2 + 2 * K


def test_full_block_does_not_carry():
    # 127 tokens in one block all picking expert 5 at every layer: cell value 127,
    # neighbouring cells (experts 4 and 6, sharing the 32-bit word) stay untouched.
    G.say("case: one block of 127 tokens on the same expert (cell 127, no carry)")
    L, E, K, T = 3, 16, 2, 127
    ids = np.empty((L, T, K), np.int32)
    ids[:, :, 0] = 5
    ids[:, :, 1] = 6
    c = Cache(2, L, E)
    c.capture(ids, np.ones(T, np.int32))
    c.check("full block")
    got = c.sig.cpu().numpy()
    assert (got[1, :, 5] == 127).all() and (got[1, :, 4] == 0).all() and (got[1, :, 7] == 0).all()


def test_request_counts_many_requests_ragged_tables():
    G.say("case: request counts for 70 requests, ragged tables with invalid entries")
    L, E = 9, 128
    rng = np.random.default_rng(10)
    c = Cache(50, L, E)
    ids = synth.prefill_picks(L, 700, E, 8, seed=11)
    c.capture(ids, rng.integers(0, 50, 700).astype(np.int32))
    tables = [list(rng.integers(-3, 53, rng.integers(0, 12))) for _ in range(70)]
    got = c.request_counts(tables)
    for r, t in enumerate(tables):
        valid = [b for b in t if 0 <= b < 50]
        assert np.array_equal(got[r], SO.request_counts(c.ref, valid)), r


@pytest.mark.parametrize("L,E,offset", [(3, 20, 0), (9, 128, 4), (6, 64, 0)])
def test_request_counts_load_paths(L, E, offset):
    # Rows of 15 words (not whole 16-byte pieces) and a cache 4 bytes off
    # 16-byte alignment take the word-by-word reads; tables of up to 150
    # blocks take several groups of 64 with a ragged last one.
    G.say(f"case: request counts, L={L} E={E}, cache offset {offset} bytes, tables of 0..150 blocks")
    nb, T = 40, 500
    rng = np.random.default_rng(20 + L)
    ids = synth.prefill_picks(L, T, E, 8, seed=21 + L)
    tb = rng.integers(0, nb, T).astype(np.int32)
    ref, _ = SO.capture(SO.new_cache(nb, L, E), ids, tb)
    flat = torch.zeros(nb * L * E + 16, dtype=torch.int8, device="cuda")
    sig = flat[offset:offset + nb * L * E].view(nb, L, E)
    B.moe_sig_capture(dev(ids), dev(tb), 0, L, E, sig)
    torch.cuda.synchronize()
    assert np.array_equal(sig.cpu().numpy().astype(np.int64), ref)
    sizes = (150, 64, 65, 1, 0, 129, 17)
    tables = [list(rng.integers(-2, nb + 2, n)) for n in sizes]
    table = np.full((len(sizes), max(sizes)), -1, np.int32)
    for r, t in enumerate(tables):
        table[r, :len(t)] = t
    out = B.moe_sig_request_counts(sig, dev(table), dev(np.array(sizes, np.int32)))
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.int64)
    for r, t in enumerate(tables):
        valid = [b for b in t if 0 <= b < nb]
        assert np.array_equal(got[r], SO.request_counts(ref, valid)), (r, len(t))


def test_empty_calls_are_no_ops():
    G.say("case: signature calls with nothing to do")
    c = Cache(4, 2, 16)
    c.capture(np.zeros((2, 0, 2), np.int32), np.zeros(0, np.int32))
    c.capture(np.zeros((0, 5, 2), np.int32), np.zeros(5, np.int32))
    B.moe_sig_reset(torch.zeros(0, dtype=torch.int32, device="cuda"), c.sig)
    c.check("empty")
    # requests with no blocks, and a cache with no blocks at all: all-zero counts
    assert not c.request_counts([[], [], []]).any()
    empty = torch.zeros((0, 2, 16), dtype=torch.int8, device="cuda")
    out = B.moe_sig_request_counts(empty, dev(np.array([[0, 1]], np.int32)), dev(np.array([2], np.int32)))
    torch.cuda.synchronize()
    assert out.shape == (1, 2, 16) and not out.cpu().numpy().any()


def test_graph_replay_of_capture_and_counts():
    # capture + request counts recorded once in a HIP graph and replayed: each
    # replay adds the same picks again, with eager work between replays.
    G.say("case: signature capture and request counts replayed from a HIP graph")
    L, E, K, T = 4, 64, 8, 96
    ids = dev(synth.prefill_picks(L, T, E, K, seed=12))
    tb = dev((np.arange(T) // BS).astype(np.int32))
    table = dev(np.arange(T // BS, dtype=np.int32)[None, :])
    nblk = dev(np.array([T // BS], np.int32))
    sig = torch.zeros((T // BS, L, E), dtype=torch.int8, device="cuda")
    out = torch.empty((1, L, E), dtype=torch.int32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        B.moe_sig_capture(ids, tb, 0, L, E, sig)
        B.moe_sig_request_counts(sig, table, nblk, out)
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        B.moe_sig_capture(ids, tb, 0, L, E, sig)
        B.moe_sig_request_counts(sig, table, nblk, out)
    base = SO.prompt_counts(ids.cpu().numpy(), E)
    for rep in range(1, 5):  # the eager call above was the first
        g.replay()
        torch.cuda.synchronize()
        junk = torch.randn(1000, device="cuda").sum().item()  # eager work between replays
        assert np.isfinite(junk)
        assert np.array_equal(out.cpu().numpy()[0].astype(np.int64), (rep + 1) * base), rep
