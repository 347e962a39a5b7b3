"""The routed launches (buckets built inside the FFN) against the separate
calls, bit for bit.

moe_expert_ffn_routed (buckets, up and down projections in one launch) and
moe_expert_ffn_up_routed (buckets and up projection) must leave exactly what
moe_bucket followed by moe_expert_ffn_up and moe_expert_ffn_down leaves: every
bucket output (counts, offsets, perm_token, pair_pos, both halves of
union_ids, union_size), the workspace h, y and the layer output; the separate
calls are themselves checked against the oracle in the parity tests, and
moe_layer (whose default is the routed up launch) is checked against the
oracle there too.  A fourth path, moe_bucket then moe_expert_ffn (up and down in one
call), must agree as well.  The one-launch path's sync counters must be zero
after every call, and its wait must never have given up.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_00466_amd import binding as B
from paper_2607_00466_amd import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

QWEN = synth.SHAPES["qwen3_30b_a3b"]
TINY = synth.SHAPES["tiny"]

KEYS = ("counts", "offsets", "perm_token", "pair_pos", "union_ids", "union_size", "ws", "y_perm",
        "out")


def _snapshot(buf, d):
    P = d.T * d.K
    return {"counts": buf.counts.cpu().numpy(), "offsets": buf.offsets.cpu().numpy(),
            "perm_token": buf.perm_token[:P].cpu().numpy(), "pair_pos": buf.pair_pos[:P].cpu().numpy(),
            "union_ids": buf.union_ids.cpu().numpy(), "union_size": buf.union_size.cpu().numpy(),
            "ws": buf.ws.view(torch.int32).cpu().numpy(), "y_perm": buf.y_perm[:P].cpu().numpy(),
            "out": buf.out.cpu().numpy()}


def _poison(buf):
    for t in (buf.counts, buf.offsets, buf.perm_token, buf.pair_pos, buf.union_ids, buf.union_size):
        t.fill_(-7)
    buf.ws.view(torch.int32).fill_(0x7fc00000)
    buf.y_perm.fill_(float("nan"))
    buf.out.fill_(float("nan"))


PATHS = ("fused", "routed", "split", "combined")


def _check_sync(buf):
    sync = buf.sync.cpu().numpy()
    assert sync[-1] == 0, "a down band of the one-launch FFN gave up waiting for h"
    assert not sync.any(), "the one-launch FFN left its counters non-zero"


def _all_paths(layer: G.Layer, routing):
    """The layer by each FFN path of moe_layer, and by moe_bucket +
    moe_expert_ffn; returns the snapshots in PATHS order."""
    d, buf = layer.d, layer.buf
    r = None
    if routing is not None:
        r = (torch.from_numpy(np.ascontiguousarray(routing[0], np.int32)).cuda(),
             torch.from_numpy(np.ascontiguousarray(routing[1], np.float32)).cuda())
    snaps = []
    for path in PATHS:
        _poison(buf)
        if path == "combined":
            ids, w = B._gate(layer.x, layer.wg, d, buf, r, None)
            B.moe_bucket(ids, d, buf.counts, buf.offsets, buf.perm_token, buf.pair_pos,
                         buf.union_ids, buf.union_size)
            B.moe_expert_ffn(layer.x, layer.p13, layer.p2, buf.offsets, buf.perm_token,
                             buf.union_ids, buf.union_size, d, buf.y_perm, buf.ws)
            B.moe_combine(buf.y_perm, buf.pair_pos, w, d, buf.out)
        else:
            B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r, path=path)
        torch.cuda.synchronize()
        snaps.append(_snapshot(buf, d))
        _check_sync(buf)
    return snaps


def _assert_equal(snaps, valid=True):
    a = snaps[0]
    for b in snaps[1:]:
        for k in KEYS:
            if not valid and k in ("perm_token", "pair_pos", "ws", "y_perm", "out"):
                continue  # not written for invalid routing (the poison stays)
            assert np.array_equal(a[k], b[k], equal_nan=True), k


@pytest.mark.parametrize("T", [1, 5, 16, 17, 33, 64])
def test_routed_equals_separate_gate_routed(T):
    G.say(f"case: routed vs separate calls, qwen shape T={T}, gate-routed")
    layer = G.Layer(QWEN, T, seed=60 + T, experts_on_host=False)
    snaps = _all_paths(layer, None)
    _assert_equal(snaps)
    G.say(f"  union {int(snaps[0]['union_size'][0])}")


@pytest.mark.parametrize("U", [16, 32, 128])
def test_routed_equals_separate_controlled(U):
    G.say(f"case: routed vs separate calls, qwen shape T=64, controlled union U={U}")
    layer = G.Layer(QWEN, 64, seed=70, experts_on_host=False)
    ids, w, _ = synth.controlled_routing(64, QWEN.E, QWEN.K, U, seed=U)
    _assert_equal(_all_paths(layer, (ids, w)))


@pytest.mark.parametrize("name,E,K,H,I,T", [
    ("most_experts", 256, 8, 256, 128, 64),     # the union reaches the 4th position a lane
    ("max_pairs", 32, 16, 256, 128, 64),        # T * K = 1024, four ids a thread
    ("ragged", 13, 3, 352, 96, 21),             # short bands, E not a multiple of 8
    ("k_eq_e", 16, 16, 256, 128, 5),            # every token on every expert
    ("single", 1, 1, 256, 128, 40),
])
def test_routed_equals_separate_shapes(name, E, K, H, I, T):
    G.say(f"case: routed vs separate calls, {name} E={E} top-{K} H={H} I={I} T={T}")
    layer = G.Layer(synth.LayerShape(name, E=E, K=K, H=H, I=I), T, seed=E + T, experts_on_host=False)
    _assert_equal(_all_paths(layer, None))


def test_routed_large_batch_takes_separate_launches():
    # Above 64 tokens the routed entry points run moe_bucket and the FFN launches.
    G.say("case: routed vs separate calls, qwen shape T=65 and T=128, controlled U=32")
    for T in (65, 128):
        layer = G.Layer(QWEN, T, seed=80, experts_on_host=False)
        ids, w, _ = synth.controlled_routing(T, QWEN.E, QWEN.K, 32, seed=T)
        _assert_equal(_all_paths(layer, (ids, w)))


def test_routed_invalid_routing():
    G.say("case: routed vs separate calls, a repeated id and an id out of range")
    layer = G.Layer(TINY, 4, seed=3, experts_on_host=False)
    w = np.full((4, 2), 0.5, np.float32)
    for ids in (np.array([[1, 1], [2, 3], [4, 5], [6, 7]], np.int32),
                np.array([[1, 16], [2, 3], [4, 5], [6, 7]], np.int32),
                np.array([[-1, 2], [2, 3], [4, 5], [6, 7]], np.int32)):
        snaps = _all_paths(layer, (ids, w))
        assert int(snaps[0]["union_size"][0]) == -1
        _assert_equal(snaps, valid=False)
        assert np.isnan(snaps[0]["y_perm"]).all(), "the FFN wrote outputs for invalid routing"


def test_routed_empty_batch():
    G.say("case: routed up launch with T = 0")
    d = B.dims(0, TINY.H, TINY.E, TINY.K, TINY.I)
    buf = B.LayerBuffers.allocate(d)
    buf.union_size.fill_(77)
    buf.counts.fill_(5)
    w13, _ = B.pack_expert_weights(*synth.expert_weights(TINY, device="cuda"))
    B.moe_expert_ffn_up_routed(torch.empty((0, TINY.H), device="cuda"), w13,
                               torch.empty((0, TINY.K), dtype=torch.int32, device="cuda"), d,
                               buf.counts, buf.offsets, buf.perm_token, buf.pair_pos, buf.union_ids,
                               buf.union_size, buf.ws)
    torch.cuda.synchronize()
    assert int(buf.union_size.item()) == 0
    assert int(buf.counts.abs().sum().item()) == 0
    assert bool((buf.union_ids == -1).all())


@pytest.mark.parametrize("T", [8, 24, 64, 65])
def test_routed_mxfp4_equals_separate(T):
    G.say(f"case: MXFP4 routed vs separate calls, E=16 top-4 H=640 I=320 T={T}, gate-routed")
    sh = synth.LayerShape("mx_routed", E=16, K=4, H=640, I=320)
    x = torch.from_numpy(synth.hidden_states(T, sh.H, T)).cuda()
    wg = torch.from_numpy(synth.gate_weights(sh, T)).cuda()
    q = synth.mxfp4_expert_weights(sh, T, device="cuda")
    up, down = B.pack_mxfp4_expert_weights(q["w1"], q["w3"], q["w2"])
    d = B.dims(T, sh.H, sh.E, sh.K, sh.I)
    buf = B.LayerBuffers.allocate(d)
    snaps = []
    for path in B.FFN_PATHS:
        _poison(buf)
        B.moe_layer_mxfp4(x, wg, up, down, d, buf, path=path)
        torch.cuda.synchronize()
        snaps.append(_snapshot(buf, d))
        _check_sync(buf)
    _assert_equal(snaps)


def test_fused_back_to_back_calls():
    # Twelve one-launch layers queued without a host synchronisation between
    # them, over changing routings and union sizes on one sync buffer: each
    # launch finds the counters its predecessor reset, and each result equals
    # the separate calls' on the same routing.
    G.say("case: one-launch FFN, 12 back-to-back calls on one sync buffer, qwen shape T=64")
    layer = G.Layer(QWEN, 64, seed=91, experts_on_host=False)
    d, buf = layer.d, layer.buf
    routings = []
    for i, U in enumerate((16, 128, 32, 64, 8, 127, 96, 24, 40, 128, 16, 72)):
        ids, w, _ = synth.controlled_routing(64, QWEN.E, QWEN.K, U, seed=100 + i)
        routings.append((torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda()))
    outs = []
    for r in routings:
        B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r)
        outs.append((buf.y_perm[:d.T * d.K].clone(), buf.out.clone()))
    torch.cuda.synchronize()
    _check_sync(buf)
    for i, r in enumerate(routings):
        B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r, path="split")
        torch.cuda.synchronize()
        assert torch.equal(outs[i][0], buf.y_perm[:d.T * d.K]), f"y_perm of call {i}"
        assert torch.equal(outs[i][1], buf.out), f"out of call {i}"


def test_fused_entry_point_checks():
    # A null or misaligned sync buffer is refused before any launch; T = 0
    # and T > 64 leave the buffer untouched.
    G.say("case: one-launch FFN argument checks, tiny shape")
    layer = G.Layer(TINY, 4, seed=5, experts_on_host=False)
    d, buf = layer.d, layer.buf
    ids, w = B._gate(layer.x, layer.wg, d, buf, None, None)
    lib = B.load()
    args = [B._ptr(layer.x), B._ptr(layer.p13), B._ptr(layer.p2), B._ptr(ids), d,
            B._ptr(buf.counts), B._ptr(buf.offsets), B._ptr(buf.perm_token), B._ptr(buf.pair_pos),
            B._ptr(buf.union_ids), B._ptr(buf.union_size), B._ptr(buf.y_perm), B._ptr(buf.ws),
            buf.ws.numel() * 4]
    assert lib.moe_expert_ffn_routed(*args, None, None) == B.MOE_ERR_INVALID
    spare = torch.zeros(2 * d.E + 2, dtype=torch.int32, device="cuda")
    misaligned = ctypes.c_void_p(spare.data_ptr() + 2)
    assert lib.moe_expert_ffn_routed(*args, misaligned, None) == B.MOE_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert not spare.any()


def test_fused_graph_replays():
    # The one-launch FFN captured in a HIP graph: its sync counters carry over
    # from replay to replay, so every replay (with eager work between) must
    # equal the eager result, leave the counters zero, and follow new routing
    # written in place.
    G.say("case: one-launch FFN in a HIP graph, qwen shape T=64, controlled U=32 then U=96")
    layer = G.Layer(QWEN, 64, seed=240, experts_on_host=False)
    d, buf = layer.d, layer.buf
    ids, w, _ = synth.controlled_routing(64, QWEN.E, QWEN.K, 32, seed=7)
    r = (torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda())
    run = lambda: B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r,  # noqa: E731
                              path="fused")
    run()
    torch.cuda.synchronize()
    eager = buf.out.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    for rep in range(4):
        buf.out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf.out, eager), f"replay {rep}"
        _check_sync(buf)
        scratch = torch.randn(2048, device="cuda").sum()  # unrelated eager work between replays
        torch.cuda.synchronize()
        del scratch
    ids2, w2, _ = synth.controlled_routing(64, QWEN.E, QWEN.K, 96, seed=8)
    r[0].copy_(torch.from_numpy(ids2))
    r[1].copy_(torch.from_numpy(w2))
    B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r, path="split")
    torch.cuda.synchronize()
    eager2 = buf.out.clone()
    buf.out.zero_()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(buf.out, eager2)
    assert not torch.equal(eager, eager2)
    _check_sync(buf)
