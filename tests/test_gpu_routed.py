"""The routed up launch (buckets built inside the up projection) against the
separate calls, bit for bit.

moe_expert_ffn_up_routed must leave exactly what moe_bucket followed by
moe_expert_ffn_up leaves: every bucket output (counts, offsets, perm_token,
pair_pos, both halves of union_ids, union_size) and the workspace h, and so
the same y and layer output; the separate calls are themselves checked
against the oracle in the parity tests, and moe_layer (which takes the routed
launch) is checked against the oracle there too.  The third path,
moe_bucket then moe_expert_ffn (up and down in one call), must agree as well.
"""
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


def _three_paths(layer: G.Layer, routing):
    """The layer by the routed launch, by moe_bucket + moe_expert_ffn_up/down, and
    by moe_bucket + moe_expert_ffn; returns the three snapshots."""
    d, buf = layer.d, layer.buf
    r = None
    if routing is not None:
        r = (torch.from_numpy(np.ascontiguousarray(routing[0], np.int32)).cuda(),
             torch.from_numpy(np.ascontiguousarray(routing[1], np.float32)).cuda())
    snaps = []
    for path in ("routed", "separate", "combined"):
        _poison(buf)
        if path == "combined":
            ids, w = B._gate(layer.x, layer.wg, d, buf, r, None)
            B.moe_bucket(ids, d, buf.counts, buf.offsets, buf.perm_token, buf.pair_pos,
                         buf.union_ids, buf.union_size)
            B.moe_expert_ffn(layer.x, layer.p13, layer.p2, buf.offsets, buf.perm_token,
                             buf.union_ids, buf.union_size, d, buf.y_perm, buf.ws)
            B.moe_combine(buf.y_perm, buf.pair_pos, w, d, buf.out)
        else:
            B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r,
                        fused=path == "routed")
        torch.cuda.synchronize()
        snaps.append(_snapshot(buf, d))
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
    snaps = _three_paths(layer, None)
    _assert_equal(snaps)
    G.say(f"  union {int(snaps[0]['union_size'][0])}")


@pytest.mark.parametrize("U", [16, 32, 128])
def test_routed_equals_separate_controlled(U):
    G.say(f"case: routed vs separate calls, qwen shape T=64, controlled union U={U}")
    layer = G.Layer(QWEN, 64, seed=70, experts_on_host=False)
    ids, w, _ = synth.controlled_routing(64, QWEN.E, QWEN.K, U, seed=U)
    _assert_equal(_three_paths(layer, (ids, w)))


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
    _assert_equal(_three_paths(layer, None))


def test_routed_large_batch_takes_two_launches():
    # Above 64 tokens the routed entry point runs moe_bucket and the up launch.
    G.say("case: routed vs separate calls, qwen shape T=65 and T=128, controlled U=32")
    for T in (65, 128):
        layer = G.Layer(QWEN, T, seed=80, experts_on_host=False)
        ids, w, _ = synth.controlled_routing(T, QWEN.E, QWEN.K, 32, seed=T)
        _assert_equal(_three_paths(layer, (ids, w)))


def test_routed_invalid_routing():
    G.say("case: routed vs separate calls, a repeated id and an id out of range")
    layer = G.Layer(TINY, 4, seed=3, experts_on_host=False)
    w = np.full((4, 2), 0.5, np.float32)
    for ids in (np.array([[1, 1], [2, 3], [4, 5], [6, 7]], np.int32),
                np.array([[1, 16], [2, 3], [4, 5], [6, 7]], np.int32),
                np.array([[-1, 2], [2, 3], [4, 5], [6, 7]], np.int32)):
        snaps = _three_paths(layer, (ids, w))
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


@pytest.mark.parametrize("T", [8, 24, 64])
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
    for fused in (True, False):
        _poison(buf)
        B.moe_layer_mxfp4(x, wg, up, down, d, buf, fused=fused)
        torch.cuda.synchronize()
        snaps.append(_snapshot(buf, d))
    _assert_equal(snaps)
