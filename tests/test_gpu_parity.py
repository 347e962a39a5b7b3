"""GPU parity: every stage of the HIP path against the CPU oracle.

Each stage is compared with the oracle stage run on the GPU's own upstream
output (ids for the buckets, buckets for the FFN), so integer outputs are
compared bit-exactly even when a near-tie (logit gap < 1e-5) lets the GPU
pick a different expert; the end-to-end output is compared only for tokens
whose selection is not a near-tie.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2607_00466_amd import binding as B
from paper_2607_00466_amd import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

TINY = synth.SHAPES["tiny"]
QWEN = synth.SHAPES["qwen3_30b_a3b"]
GPTOSS = synth.SHAPES["gpt_oss_120b"]


@pytest.fixture(scope="module")
def qwen_layer():
    G.say("building the qwen3_30b_a3b-shaped layer (E=128 top-8 H=2048 I=768), T=64")
    return G.Layer(QWEN, 64)


def _full_check(layer: G.Layer, g: dict, routed_by_gate: bool, routing=None) -> None:
    s = layer.shape
    w1, w3, w2 = layer.host_weights()
    if routed_by_gate:
        near = G.check_gate(g, layer.x_np, layer.wg_np, s.K)
        ids, wts = g["ids"].astype(np.int64), g["weights"]
    else:
        near = np.zeros(layer.T, dtype=bool)
        ids, wts = routing
    G.compare_buckets(g, ids, s.E)
    b = O.bucket(ids, s.E)
    y = O.expert_ffn(layer.x_np, w1, w3, w2, ids, b)
    G.check_output(g["y_slots"], y, "expert FFN per slot")
    out = O.combine(y, b["pair_pos"], np.asarray(wts, np.float64))
    G.check_output(g["out"], out, "layer output (GPU routing)")
    if routed_by_gate:
        ok = ~near
        logits = O.gate_logits(layer.x_np, layer.wg_np)
        ref_ids = O.select_experts(logits, s.K)
        if np.array_equal(ref_ids, g["ids"]):
            # the oracle routes exactly as the GPU did, so its slot outputs are
            # the ones above; only the oracle's own weights remain to apply
            ref_out = O.combine(y, b["pair_pos"], O.routing_weights(logits, ref_ids))
        else:
            ref_out = O.moe_layer(layer.x_np, layer.wg_np, w1, w3, w2, s.K)["out"]
        G.check_output(g["out"][ok], ref_out[ok], "layer output vs oracle end to end")


def test_tiny_layer_end_to_end():
    G.say("case: tiny layer E=16 top-2 H=256 I=128 T=8 seed 0, gate-routed")
    layer = G.Layer(TINY, 8)
    g = layer.run()
    _full_check(layer, g, True)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_tiny_layer_seeds(seed):
    G.say(f"case: tiny layer seed {seed}, T=40 (ragged token tiles)")
    layer = G.Layer(TINY, 40, seed=seed)
    _full_check(layer, layer.run(), True)


def test_qwen_layer_gate_routed(qwen_layer):
    G.say("case: qwen layer gate-routed T=64")
    g = qwen_layer.run()
    G.say(f"  union size {g['union_size']}, max bucket {g['counts'].max()}")
    _full_check(qwen_layer, g, True)


@pytest.mark.parametrize("U", [16, 32, 64, 96, 128])
def test_qwen_controlled_union(qwen_layer, U):
    G.say(f"case: qwen layer, gate bypassed, controlled union U={U}, T=64")
    ids, w, _ = synth.controlled_routing(64, QWEN.E, QWEN.K, U, seed=0)
    g = qwen_layer.run(routing=(ids, w))
    assert g["union_size"] == len(set(ids.ravel().tolist()))
    _full_check(qwen_layer, g, False, routing=(ids.astype(np.int64), w))


@pytest.mark.parametrize("T", [1, 8, 16, 17, 32, 128, 256])
def test_qwen_batch_sweep(T):
    G.say(f"case: qwen layer, controlled union U=32, batch T={T}")
    layer = G.Layer(QWEN, T)
    ids, w, _ = synth.controlled_routing(T, QWEN.E, QWEN.K, 32, seed=T)
    g = layer.run(routing=(ids, w))
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


def test_bucket_over_64_tokens_takes_groups():
    # Every token picks the same 8 experts: 200 tokens per bucket, four token groups.
    G.say("case: qwen layer, T=200, all tokens on experts 0..7 (buckets of 200)")
    layer = G.Layer(QWEN, 200)
    ids = np.tile(np.arange(8, dtype=np.int32), (200, 1))
    w = np.full((200, 8), 1 / 8, np.float32)
    g = layer.run(routing=(ids, w))
    assert g["union_size"] == 8
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


def test_heavy_experts_on_one_xcd():
    # Union = experts 0..31; experts 0, 8, 16, 24 (union positions of one XCD)
    # take every token, so that XCD has more (band, token group) items than
    # workgroup slots and its slots loop.
    shape = synth.LayerShape("heavy_xcd", E=32, K=8, H=512, I=256)
    T = 512
    G.say(f"case: E=32 top-8 H=512 I=256 T={T}, experts 0/8/16/24 take all {T} tokens")
    rng = np.random.default_rng(11)
    heavy = np.array([0, 8, 16, 24], np.int32)
    light = np.setdiff1d(np.arange(32, dtype=np.int32), heavy)
    ids = np.empty((T, 8), np.int32)
    for t in range(T):
        ids[t, :4] = heavy
        ids[t, 4:] = rng.choice(light, 4, replace=False)
    w = rng.dirichlet(np.ones(8), size=T).astype(np.float32)
    layer = G.Layer(shape, T, seed=12)
    g = layer.run(routing=(ids, w))
    assert g["union_size"] == 32
    assert g["counts"][heavy].tolist() == [T] * 4
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


@pytest.mark.parametrize("T", [64, 100])
def test_most_experts(T):
    # E = 256, the most the library takes: the union reaches the last of the
    # four union positions a lane holds in the FFN's lookup.  T = 64 takes the
    # small-batch kernels, T = 100 the large-batch ones (whose buckets all fit
    # one 128-token group here, so they too deal whole experts).
    G.say(f"case: E=256 top-8 H=256 I=128 T={T}, gate-routed")
    shape = synth.LayerShape("most_experts", E=256, K=8, H=256, I=128)
    layer = G.Layer(shape, T, seed=30 + T)
    g = layer.run()
    assert g["union_size"] > 192
    _full_check(layer, g, True)


def test_most_experts_heavy_buckets():
    # E = 256 with experts 250..253 in every token (three token groups each,
    # first in dispatch order) beside an almost full union of light experts.
    shape = synth.LayerShape("most_experts_heavy", E=256, K=8, H=256, I=128)
    T = 200
    G.say(f"case: E=256 top-8 H=256 I=128 T={T}, experts 250..253 take every token")
    rng = np.random.default_rng(13)
    heavy = np.array([250, 251, 252, 253], np.int32)
    light = np.setdiff1d(np.arange(256, dtype=np.int32), heavy)
    ids = np.empty((T, 8), np.int32)
    for t in range(T):
        ids[t, :4] = heavy
        ids[t, 4:] = rng.choice(light, 4, replace=False)
    w = rng.dirichlet(np.ones(8), size=T).astype(np.float32)
    layer = G.Layer(shape, T, seed=14)
    g = layer.run(routing=(ids, w))
    assert g["union_size"] > 192
    assert g["counts"][heavy].tolist() == [T] * 4
    assert g["union_ids"][256:260].tolist() == heavy.tolist()  # first in dispatch order
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


@pytest.mark.parametrize("n", [128, 129])
def test_large_batch_dealing_boundary(n):
    # Batches over 64 tokens deal whole experts over the XCDs while every
    # bucket fits one 128-token group, and (expert, band) units once one does
    # not: a bucket of 128 tokens takes the first, 129 the second.
    G.say(f"case: qwen layer T=160, expert 3 takes {n} tokens, the others light")
    T = 160
    ids, w = G.fixed_bucket_routing(T, QWEN.E, QWEN.K, [(3, n)], seed=n)
    layer = G.Layer(QWEN, T, seed=15)
    g = layer.run(routing=(ids, w))
    assert int(g["counts"][3]) == n and int(g["counts"].max()) == n
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


@pytest.mark.parametrize("T", [21, 203])
def test_ragged_shape_partial_bands(T):
    # H and I multiples of 32 but not of the 64/128-row bands; E not a multiple of
    # 8.  T = 203 takes the large-batch kernels and the gate's 8 x 8 tiles, with a
    # partial last tile of experts and of tokens.
    G.say(f"case: ragged shape E=13 top-3 H=352 I=96 T={T}")
    shape = synth.LayerShape("ragged", E=13, K=3, H=352, I=96)
    layer = G.Layer(shape, T, seed=4)
    _full_check(layer, layer.run(), True)


def test_ragged_shape_even_steps_short_band():
    # H = 320 (an even number of k-steps, 2.5 bands of W2) and I = 96 (a short
    # last band of W1/W3), E not a multiple of 8, a 2-tile kernel (T = 21).
    G.say("case: ragged shape E=13 top-3 H=320 I=96 T=21")
    shape = synth.LayerShape("ragged_even", E=13, K=3, H=320, I=96)
    layer = G.Layer(shape, 21, seed=6)
    _full_check(layer, layer.run(), True)


def test_k_equals_e():
    G.say("case: K = E = 16, H=256 I=128 T=5")
    shape = synth.LayerShape("k_eq_e", E=16, K=16, H=256, I=128)
    layer = G.Layer(shape, 5, seed=6)
    g = layer.run()
    assert g["union_size"] == 16
    _full_check(layer, g, True)


@pytest.mark.parametrize("T", [5, 70, 200])
def test_single_expert(T):
    # E = K = 1: every token on expert 0 with weight 1, a union of one.  T = 70
    # takes the large-batch kernels with one 128-token group; T = 200 two groups,
    # and the gate's 8 x 8 tiles with one live expert each.
    G.say(f"case: E=1 top-1 H=256 I=128 T={T}, gate-routed")
    shape = synth.LayerShape("single_expert", E=1, K=1, H=256, I=128)
    layer = G.Layer(shape, T, seed=40 + T)
    g = layer.run()
    assert g["union_size"] == 1
    assert g["counts"].tolist() == [T]
    assert np.all(g["weights"] == 1.0)
    _full_check(layer, g, True)


def test_duplicate_gate_rows_tie_to_lower_id():
    G.say("case: gate rows 3 and 11 identical (exact ties), tiny shape T=64")
    layer = G.Layer(TINY, 64, seed=9)
    layer.wg_np = layer.wg_np.copy()
    layer.wg_np[11] = layer.wg_np[3]
    layer.wg = torch.from_numpy(layer.wg_np).cuda()
    g = layer.run()
    assert np.array_equal(g["logits"][:, 3], g["logits"][:, 11])
    for row in g["ids"].tolist():
        if 11 in row:
            assert 3 in row and row.index(3) < row.index(11)
    assert any(3 in row and 11 not in row for row in g["ids"].tolist())
    _full_check(layer, g, True)


def _gate(x: np.ndarray, wg: torch.Tensor, shape) -> tuple:
    T = x.shape[0]
    d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
    logits = torch.empty((T, shape.E), device="cuda")
    ids = torch.empty((T, shape.K), dtype=torch.int32, device="cuda")
    wts = torch.empty((T, shape.K), device="cuda")
    B.moe_gate_topk(torch.from_numpy(x).cuda(), wg, d, logits, ids, wts)
    torch.cuda.synchronize()
    return logits.cpu().numpy(), ids.cpu().numpy(), wts.cpu().numpy()


@pytest.mark.parametrize("shape", [QWEN, GPTOSS], ids=lambda s: s.name)
def test_gate_scores_do_not_depend_on_the_batch(shape):
    """A token's logits, picks and weights are the same bits in any batch: the
    batch decides the tile shape of the score kernel (4 x 4 up to 128 tokens,
    8 x 8 above), not the reduction order of a score."""
    G.say(f"case: gate of a 640-token batch vs sub-batches of 1..129 tokens, {shape.name}")
    x = synth.hidden_states(640, shape.H, seed=21)
    wg_np = synth.gate_weights(shape, seed=21)
    wg_np[11] = wg_np[3]  # an exact tie inside the 8 x 8 tiles too
    wg = torch.from_numpy(wg_np).cuda()
    full = _gate(x, wg, shape)
    assert np.array_equal(full[0][:, 3], full[0][:, 11])
    for t0, t1 in [(0, 1), (0, 8), (5, 69), (100, 228), (200, 329), (3, 640)]:
        part = _gate(x[t0:t1], wg, shape)
        for name, a, b in zip(("logits", "ids", "weights"), full, part):
            assert np.array_equal(a[t0:t1], b), f"{name} of tokens {t0}..{t1 - 1} differ"
    G.check_gate({"logits": full[0], "ids": full[1], "weights": full[2]}, x, wg_np, shape.K)


@pytest.mark.parametrize("path", B.FFN_PATHS)
def test_layer_output_does_not_depend_on_the_batch(path):
    """A token's gate output and layer output are the same bits whatever else is
    in its batch: sub-batches on both sides of the 64-token kernel switch and
    of the 128-token group give the rows of the full batch's result."""
    G.say(f"case: qwen layer, 256-token batch vs sub-batches of 1..253 tokens, path {path}")
    layer = G.Layer(QWEN, 256, seed=23, experts_on_host=False)
    full = layer.run(path=path)
    for t0, t1 in [(0, 1), (0, 16), (16, 80), (100, 164), (0, 65), (80, 209), (3, 256)]:
        d = B.dims(t1 - t0, QWEN.H, QWEN.E, QWEN.K, QWEN.I)
        buf = B.LayerBuffers.allocate(d)
        B.moe_layer(layer.x[t0:t1].contiguous(), layer.wg, layer.p13, layer.p2, d, buf, path=path)
        torch.cuda.synchronize()
        part = G.fetch(buf, d)
        for k in ("logits", "ids", "weights", "out"):
            assert np.array_equal(full[k][t0:t1], part[k]), f"{k} of tokens {t0}..{t1 - 1} differ"


def test_zero_input():
    G.say("case: x = 0 (all logits 0): ids 0..K-1, weights 1/K, output 0")
    layer = G.Layer(TINY, 8)
    layer.x.zero_()
    layer.x_np = np.zeros_like(layer.x_np)
    g = layer.run()
    assert np.array_equal(g["ids"], np.tile(np.arange(TINY.K), (8, 1)))
    assert np.all(g["weights"] == np.float32(1.0 / TINY.K))
    assert np.all(g["out"] == 0)


def test_empty_batch():
    G.say("case: T = 0")
    d = B.dims(0, TINY.H, TINY.E, TINY.K, TINY.I)
    buf = B.LayerBuffers.allocate(d)
    buf.union_size.fill_(77)
    buf.counts.fill_(5)
    x = torch.empty((0, TINY.H), device="cuda")
    w13, w2 = B.pack_expert_weights(*synth.expert_weights(TINY, device="cuda"))
    B.moe_layer(x, torch.zeros((TINY.E, TINY.H), device="cuda"), w13, w2, d, buf)
    torch.cuda.synchronize()
    assert int(buf.union_size.item()) == 0
    assert int(buf.counts.abs().sum().item()) == 0
    assert int(buf.offsets.abs().sum().item()) == 0
    assert bool((buf.union_ids == -1).all())


def test_invalid_routing_flags_union():
    G.say("case: repeated id within a token -> union_size = -1, FFN does nothing")
    layer = G.Layer(TINY, 4)
    ids = np.array([[1, 1], [2, 3], [4, 5], [6, 7]], np.int32)
    w = np.full((4, 2), 0.5, np.float32)
    layer.buf.y_perm.fill_(123.0)
    g = layer.run(routing=(ids, w))
    assert g["union_size"] == -1
    assert np.all(g["y_slots"] == 123.0)
    ids2 = np.array([[1, 16], [2, 3], [4, 5], [6, 7]], np.int32)  # out of range
    g = layer.run(routing=(ids2, w))
    assert g["union_size"] == -1


def test_invalid_routing_over_64_tokens():
    # The same flag when the batch takes the kernels that deal (expert, band)
    # units over the XCDs: they read no union entry and write nothing.
    T = 100
    G.say(f"case: repeated id within a token, T={T} -> union_size = -1, FFN does nothing")
    layer = G.Layer(TINY, T)
    rng = np.random.default_rng(21)
    ids = np.stack([rng.choice(TINY.E, TINY.K, replace=False) for _ in range(T)]).astype(np.int32)
    ids[57] = [9, 9]
    w = np.full((T, TINY.K), 0.5, np.float32)
    layer.buf.y_perm.fill_(123.0)
    g = layer.run(routing=(ids, w))
    assert g["union_size"] == -1
    assert np.all(g["y_slots"] == 123.0)


@pytest.mark.parametrize("T,E", [(4096, 128), (2048, 256)])
def test_bucket_large_batch(T, E):
    # Both fill the 16384-word bitmap limit (LDS above 64 KiB); E = 256 also
    # ranks each expert with two threads instead of four.
    G.say(f"case: bucket only, T={T} E={E} K=8 (bitmap limit)")
    K = 8
    rng = np.random.default_rng(5 + E)
    ids = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    d = B.dims(T, 64, E, K, 32)
    buf = B.LayerBuffers.allocate(d)
    B.moe_bucket(torch.from_numpy(ids).cuda(), d, buf.counts, buf.offsets, buf.perm_token,
                 buf.pair_pos, buf.union_ids, buf.union_size)
    torch.cuda.synchronize()
    G.compare_buckets(G.fetch(buf, d), ids.astype(np.int64), E)


@pytest.mark.parametrize("H,I,T", [(B.MOE_MAX_H, 256, 24), (256, B.MOE_MAX_I, 24),
                                   (B.MOE_MAX_H, 256, 80), (256, B.MOE_MAX_I, 80)])
def test_largest_hidden_and_intermediate(H, I, T):
    # The limits on H and I: 512-step reductions and 128 or 256 row bands an
    # expert, through the routed launch (T <= 64) and the large-batch kernels
    # (T > 64, one bucket of 80 tokens in a 128-token pass).
    sh = synth.LayerShape("max_hi", E=4, K=2, H=H, I=I)
    G.say(f"case: E=4 top-2 H={H} I={I} T={T}, expert 1 takes every token")
    layer = G.Layer(sh, T, seed=(H + I + T) % 1000)
    ids, w = G.fixed_bucket_routing(T, sh.E, sh.K, [(1, T)], seed=T)
    g = layer.run(routing=(ids, w))
    assert int(g["counts"][1]) == T
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


def test_largest_batch_gate_routed():
    # The limit on T: 4096 tokens x top-8, gate-routed end to end (buckets of
    # about 256 tokens, two or more 128-token groups each).
    sh = synth.LayerShape("max_t", E=128, K=8, H=256, I=128)
    T = B.MOE_MAX_T
    G.say(f"case: E=128 top-8 H=256 I=128 T={T}, gate-routed")
    layer = G.Layer(sh, T, seed=3)
    g = layer.run()
    assert int(g["counts"].max()) > 128
    _full_check(layer, g, True)


def test_union_dispatch_order_at_tile_boundaries():
    # One pick per token, so each expert's count is set exactly: 15, 16 and 17
    # tokens straddle the first 16-token tile, 32/33 the second, 48/49 the
    # third; experts 6 and 11 take none.  Dispatch order: more tiles first,
    # equal tiles by ascending id.
    E = 12
    counts = [15, 16, 17, 32, 33, 1, 0, 16, 48, 49, 2, 0]
    ids = np.repeat(np.arange(E, dtype=np.int32), counts)
    np.random.default_rng(8).shuffle(ids)
    T = ids.size
    G.say(f"case: bucket only, T={T} E={E} K=1, counts {counts}")
    d = B.dims(T, 64, E, 1, 32)
    buf = B.LayerBuffers.allocate(d)
    B.moe_bucket(torch.from_numpy(ids.reshape(T, 1)).cuda(), d, buf.counts, buf.offsets,
                 buf.perm_token, buf.pair_pos, buf.union_ids, buf.union_size)
    torch.cuda.synchronize()
    g = G.fetch(buf, d)
    assert g["union_size"] == 10
    assert g["union_ids"][:E].tolist() == [0, 1, 2, 3, 4, 5, 7, 8, 9, 10, -1, -1]
    assert g["union_ids"][E:].tolist() == [9, 4, 8, 2, 3, 0, 1, 5, 7, 10, -1, -1]
    G.compare_buckets(g, ids.reshape(T, 1).astype(np.int64), E)


def test_combine_alone():
    G.say("case: combine on oracle slot outputs, qwen shape T=64")
    T, E, K, H = 64, 128, 8, 2048
    ids, w, _ = synth.controlled_routing(T, E, K, 48, seed=3)
    b = O.bucket(ids.astype(np.int64), E)
    rng = np.random.default_rng(8)
    y = rng.standard_normal((T * K, H)).astype(np.float32)
    d = B.dims(T, H, E, K, 768)
    out = torch.empty((T, H), device="cuda")
    B.moe_combine(torch.from_numpy(y).cuda(), torch.from_numpy(b["pair_pos"].ravel().astype(np.int32)).cuda(),
                  torch.from_numpy(w).cuda(), d, out)
    torch.cuda.synchronize()
    ref = O.combine(y.astype(np.float64), b["pair_pos"], w.astype(np.float64))
    assert np.abs(out.cpu().numpy() - ref).max() <= 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("T,K,H", [(3, 2, 32), (5, 4, 288), (7, 8, 2880)])
def test_combine_ragged_rows_and_slots_out_of_range(T, K, H):
    """Hidden sizes that leave the last wave partly idle (H/4 not a multiple of
    64), and slots outside [0, T*K), which contribute nothing: the reference
    points them at an appended zero row."""
    G.say(f"case: combine alone, T={T} K={K} H={H}, some slots out of range")
    rng = np.random.default_rng(T * 100 + H)
    P = T * K
    pp = rng.permutation(P).astype(np.int32).reshape(T, K)
    pp[0, K - 1] = -1
    pp[T - 1, 0] = P
    pp[T // 2, K // 2] = 1 << 30
    w = rng.random((T, K)).astype(np.float32)
    y = rng.standard_normal((P, H)).astype(np.float32)
    d = B.dims(T, H, max(K, 8), K, 32)
    out = torch.full((T, H), float("nan"), device="cuda")
    B.moe_combine(torch.from_numpy(y).cuda(), torch.from_numpy(pp.ravel()).cuda(),
                  torch.from_numpy(w).cuda(), d, out)
    torch.cuda.synchronize()
    y_ext = np.vstack([y.astype(np.float64), np.zeros((1, H))])
    pp_ref = np.where((pp >= 0) & (pp < P), pp, P)
    ref = O.combine(y_ext, pp_ref, w.astype(np.float64))
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() <= 1e-5 * np.abs(ref).max()


def test_deterministic(qwen_layer):
    G.say("case: two runs of the qwen layer are bitwise equal")
    a = qwen_layer.run()
    b = qwen_layer.run()
    for key in ("logits", "ids", "weights", "counts", "offsets", "perm_token", "pair_pos",
                "union_ids", "y_slots", "out"):
        assert np.array_equal(a[key], b[key]), key


@pytest.fixture(scope="module")
def gpt_oss_layer():
    # Full gpt-oss shape: 6.4 GB of bf16 experts on the device and a host copy
    # of their bit patterns for the oracle.
    G.say("building the gpt-oss-shaped layer (E=128 top-4 H=I=2880, bf16 experts), T=256")
    return G.Layer(GPTOSS, 256)


def test_gpt_oss_layer_gate_routed(gpt_oss_layer):
    # Every output row and every slot row against the oracle.
    G.say("case: gpt-oss-shaped layer T=256, gate-routed, all 256 tokens and 1024 slots")
    g = gpt_oss_layer.run()
    G.say(f"  union size {g['union_size']}, max bucket {g['counts'].max()}")
    assert g["y_slots"].shape[0] == 256 * GPTOSS.K
    _full_check(gpt_oss_layer, g, True)


@pytest.mark.parametrize("U", [32, 128])
def test_gpt_oss_controlled_union(gpt_oss_layer, U):
    G.say(f"case: gpt-oss-shaped layer T=256, controlled union U={U}, all tokens and slots")
    ids, w, _ = synth.controlled_routing(256, GPTOSS.E, GPTOSS.K, U, seed=U)
    g = gpt_oss_layer.run(routing=(ids, w))
    G.say(f"  union size {g['union_size']}, max bucket {g['counts'].max()}")
    assert g["union_size"] == len(set(ids.ravel().tolist()))
    _full_check(gpt_oss_layer, g, False, routing=(ids.astype(np.int64), w))


@pytest.mark.parametrize("T,heavy", [(24, [(10, 24), (20, 17)]),
                                     (32, [(3, 17), (40, 24), (77, 32)])])
def test_two_tile_pass(T, heavy):
    # 16 < T <= 32 takes the two-tile kernel; buckets of 17, 24 and 32 tokens
    # run its two-tile pass (the other buckets, of a few tokens, its one-tile pass).
    G.say(f"case: qwen layer T={T}, buckets of {[n for _, n in heavy]} tokens (two-tile pass)")
    ids, w = G.fixed_bucket_routing(T, QWEN.E, QWEN.K, heavy, seed=T)
    layer = G.Layer(QWEN, T, seed=50 + T)
    g = layer.run(routing=(ids, w))
    assert [int(g["counts"][e]) for e, _ in heavy] == [n for _, n in heavy]
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


def test_forced_near_tie():
    # Gate rows 5 and 9 differ only by 2^-20 at hidden position 200, so
    # logit 9 - logit 5 = 2^-20 x[200]: tokens where those two compete for the
    # second of K = 2 places are near-ties by construction.  Every row is
    # otherwise one-hot, so each fp32 logit is exact or takes one rounding.
    #   t % 4 == 0, 1: x[200] = +-3, a gap of 2.9e-6 that fp32 resolves: the
    #                  GPU picks what the oracle picks;
    #   t % 4 == 2:    x[200] = +-0.1, a gap of 9.5e-8, below half an ulp of 2:
    #                  the GPU's logits tie exactly and the lower id 5 wins,
    #                  while for x[200] > 0 the oracle picks 9;
    #   t % 4 == 3:    experts 2 and 7 lead by far: no near-tie.
    T, E, H = 32, TINY.E, TINY.H
    G.say("case: tiny shape T=32, gate rows 5 and 9 a 2^-20 step apart (forced near-ties)")
    layer = G.Layer(TINY, T, seed=15)
    rng = np.random.default_rng(15)
    wg = np.zeros((E, H), np.float32)
    wg[np.arange(E), np.arange(E)] = 1.0
    wg[9, 9] = 0.0
    wg[9, 5] = 1.0
    wg[9, 200] = 2.0 ** -20
    x = rng.uniform(-0.5, 0.5, (T, H)).astype(np.float32)
    for t in range(T):
        kind = t % 4
        x[t, 2] = 4.0
        if kind < 3:
            x[t, 5] = 2.0
            mag = 3.0 if kind < 2 else 0.1
            sign = (1.0 if kind == 0 else -1.0) if kind < 2 else (1.0 if (t // 4) % 2 == 0 else -1.0)
            x[t, 200] = sign * mag
        else:
            x[t, 7] = 2.0
            x[t, 5] = -3.0
    layer.x_np, layer.wg_np = x, wg
    layer.x = torch.from_numpy(x).cuda()
    layer.wg = torch.from_numpy(wg).cuda()
    g = layer.run()
    logits = O.gate_logits(x, wg)
    near = O.selection_gaps(logits, TINY.K) < G.NEAR_TIE
    assert near.sum() == 24 and not near[3::4].any()
    ref = O.select_experts(logits, TINY.K)
    differ = [t for t in range(T) if set(ref[t].tolist()) != set(g["ids"][t].tolist())]
    G.say(f"  tokens where the GPU's valid pick differs from the oracle's: {differ}")
    assert differ == [t for t in range(2, T, 8)]  # x[200] = +0.1: the oracle picks 9, the GPU 5
    assert all(sorted(g["ids"][t].tolist()) == [2, 5] for t in differ)
    _full_check(layer, g, True)


def test_graph_replay_matches_eager():
    # The layer captured as a HIP graph (as the benchmark times it) gives the
    # eager result on every replay, with eager work and syncs in between, and
    # follows new input values written in place.
    G.say("case: qwen layer T=64 gate-routed, HIP graph replays vs eager")
    layer = G.Layer(QWEN, 64, experts_on_host=False)
    d, buf = layer.d, layer.buf
    run = lambda: B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf)  # noqa: E731
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
        scratch = torch.randn(1024, device="cuda") * 2  # unrelated eager work between replays
        torch.cuda.synchronize()
        del scratch
    x2 = torch.from_numpy(synth.hidden_states(64, QWEN.H, seed=5)).cuda()
    layer.x.copy_(x2)
    run()
    torch.cuda.synchronize()
    eager2 = buf.out.clone()
    buf.out.zero_()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(buf.out, eager2)
    assert not torch.equal(eager, eager2)


def test_graph_replay_large_batch_token_groups():
    # A domain-clustered batch of 128 tokens (the >64-token mapping: token
    # groups, heaviest experts first) captured in a graph: every replay equals
    # the eager result bit for bit, and the output matches the oracle.
    G.say("case: qwen layer T=128 domain-clustered (token groups), graph replays vs eager vs oracle")
    model = synth.DomainModel()
    subsets = synth.domain_subsets(model, 1, seed=0)
    doms = synth.domain_batches(model, 128)["same_3"]
    ids, w = synth.domain_routing(model, subsets, doms, 0, seed=0)
    layer = G.Layer(QWEN, 128, seed=9)
    g0 = layer.run(routing=(ids, w))
    assert g0["counts"].max() > 64  # some expert really has more than one token group
    _full_check(layer, g0, False, routing=(ids.astype(np.int64), w))
    d, buf = layer.d, layer.buf
    r = (torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda())
    run = lambda: B.moe_layer(layer.x, layer.wg, layer.p13, layer.p2, d, buf, routing=r)  # noqa: E731
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
        scratch = torch.randn(2048, device="cuda").sum()  # unrelated eager work between replays
        torch.cuda.synchronize()
        del scratch


def test_batch_of_65_tokens_crosses_the_group_boundary():
    # 65 tokens all on the same 8 experts: one group of 64 and one of 1.
    G.say("case: qwen layer, T=65, all tokens on experts 3..10 (two token groups each)")
    layer = G.Layer(QWEN, 65, seed=10)
    ids = np.tile(np.arange(3, 11, dtype=np.int32), (65, 1))
    w = np.random.default_rng(11).dirichlet(np.ones(8), size=65).astype(np.float32)
    g = layer.run(routing=(ids, w))
    assert g["counts"][3:11].tolist() == [65] * 8
    _full_check(layer, g, False, routing=(ids.astype(np.int64), w))


def _band_reference(srcs, band_rows: int, wave_rows: int) -> np.ndarray:
    """The documented packed order, built band by band: per expert, band, k-step,
    wave and its two fragments, the 64 lane pieces (lane l: row l % 16, values
    8 (l // 16) .. + 7 of the k-step).  srcs: one [E, R, K] array per fragment
    kind (up: W1, W3 for fragments 0, 1) or a single array whose fragment f is
    the wave's f-th 16-row tile (down)."""
    E, R, K = srcs[0].shape
    nk = K // 32
    bands = []
    for b in range((R + band_rows - 1) // band_rows):
        waves = min(band_rows, R - b * band_rows) // wave_rows
        blk = np.empty((E, nk, waves, 2, 64, 8), np.uint16)
        for w in range(waves):
            for f in range(2):
                src = srcs[f] if len(srcs) == 2 else srcs[0]
                r0 = b * band_rows + w * wave_rows + (0 if len(srcs) == 2 else 16 * f)
                tile = src[:, r0:r0 + 16, :].reshape(E, 16, nk, 4, 8).transpose(0, 2, 3, 1, 4)
                blk[:, :, w, f] = tile.reshape(E, nk, 64, 8)
        bands.append(blk.reshape(E, -1))
    return np.concatenate(bands, axis=1).reshape(-1)


@pytest.mark.parametrize("E,I,H", [(3, 32, 32), (2, 96, 64), (128, 768, 2048), (2, 2880, 2880)])
def test_pack_weights_are_the_documented_permutation(E, I, H):
    # I = 32 and 96 and H = 2880 leave a short last band (2 of 4 waves).
    G.say(f"case: pack up and down, E={E} I={I} H={H}")
    g = torch.Generator(device="cuda")
    g.manual_seed(E * 1000 + I)
    w1, w3 = (torch.randn((E, I, H), generator=g, device="cuda").to(torch.bfloat16) for _ in range(2))
    w2 = torch.randn((E, H, I), generator=g, device="cuda").to(torch.bfloat16)
    up = synth.bf16_bits(B.moe_pack_up_weights(w1, w3))
    assert np.array_equal(up.reshape(-1), _band_reference([synth.bf16_bits(w1), synth.bf16_bits(w3)], 64, 16))
    down = synth.bf16_bits(B.moe_pack_down_weights(w2))
    assert np.array_equal(down.reshape(-1), _band_reference([synth.bf16_bits(w2)], 128, 32))


def test_stream_probe_reads_without_writing():
    # The calibration probe reads a buffer (a ragged size: not a multiple of its
    # per-workgroup stretch) and leaves the sink alone unless its checksum hits
    # the fixed constant, which all-ones data does not.
    G.say("case: streaming-read probe over 3 MiB + 48 bytes")
    buf = torch.ones((3 << 20) // 4 + 12, dtype=torch.float32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.moe_stream_read_probe(buf, sink)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
