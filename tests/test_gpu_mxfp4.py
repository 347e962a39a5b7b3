"""GPU parity of the MXFP4 expert path against the dequantizing oracle.

The MXFP4 FFN expands FP4 codes to bf16 in registers and then multiplies as
the bf16 FFN does, so besides the oracle comparison (float64 on the
dequantized weights) it must equal the bf16 path run on the dequantized
weights bit for bit.  The packed layouts are checked against the permutation
the header documents, written out here with NumPy.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from oracle import mxfp4 as MX
from paper_2607_00466_amd import binding as B
from paper_2607_00466_amd import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

GPTOSS = synth.SHAPES["gpt_oss_120b"]


class MxLayer:
    """One layer with MXFP4 experts on the device, plus host copies for the oracle."""

    def __init__(self, shape: synth.LayerShape, T: int, seed: int = 0, q=None):
        self.shape, self.T = shape, T
        self.x_np = synth.hidden_states(T, shape.H, seed)
        self.wg_np = synth.gate_weights(shape, seed)
        self.x = torch.from_numpy(self.x_np).cuda()
        self.wg = torch.from_numpy(self.wg_np).cuda()
        self.q = q if q is not None else synth.mxfp4_expert_weights(shape, seed, device="cuda")
        self.up, self.down = B.pack_mxfp4_expert_weights(self.q["w1"], self.q["w3"], self.q["w2"])
        self.d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
        self.buf = B.LayerBuffers.allocate(self.d)

    def host_q(self, experts=None):
        """{name: (codes, scales)} as NumPy, all experts or only the listed ones (others zero)."""
        out = {}
        for name, (c, s) in self.q.items():
            if experts is None:
                out[name] = (c.cpu().numpy(), s.cpu().numpy())
                continue
            hc = np.zeros(tuple(c.shape), np.uint8)
            hs = np.full(tuple(s.shape), 127, np.uint8)
            for e in experts:
                hc[e] = c[e].cpu().numpy()
                hs[e] = s[e].cpu().numpy()
            out[name] = (hc, hs)
        return out

    def run(self, routing=None):
        if routing is not None:
            routing = (torch.from_numpy(np.ascontiguousarray(routing[0], np.int32)).cuda(),
                       torch.from_numpy(np.ascontiguousarray(routing[1], np.float32)).cuda())
        B.moe_layer_mxfp4(self.x, self.wg, self.up, self.down, self.d, self.buf, routing=routing)
        torch.cuda.synchronize()
        return G.fetch(self.buf, self.d)


def _check_layer(layer: MxLayer, g: dict, routing=None) -> None:
    s = layer.shape
    if routing is None:
        G.check_gate(g, layer.x_np, layer.wg_np, s.K)
        ids, wts = g["ids"].astype(np.int64), g["weights"]
    else:
        ids, wts = routing
    G.compare_buckets(g, ids, s.E)
    q = layer.host_q()
    b = O.bucket(ids, s.E)
    y = MX.expert_ffn(layer.x_np, q["w1"], q["w3"], q["w2"], ids, b)
    G.check_output(g["y_slots"], y, "MXFP4 expert FFN per slot")
    out = O.combine(y, b["pair_pos"], np.asarray(wts, np.float64))
    G.check_output(g["out"], out, "MXFP4 layer output")


# ---------------------------------------------------------------------------- packing

def _dwords(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a).view(np.uint32)


def _wg_bands(per_band: np.ndarray) -> np.ndarray:
    """Regroup [E, wave band, slot, ...] into the packed order: per expert, groups
    of 4 wave bands (the last may hold fewer), slot, wave band within the group."""
    E, nwb = per_band.shape[:2]
    parts = [np.swapaxes(per_band[:, j:j + 4], 1, 2).reshape(E, -1) for j in range(0, nwb, 4)]
    return np.concatenate(parts, axis=1).reshape(-1)


# H = 64, 320 and 2880 leave a short last workgroup band of W2 (2 of 4 wave bands).
@pytest.mark.parametrize("E,I,H", [(3, 64, 64), (2, 192, 320), (4, 2880, 2880)])
def test_pack_mxfp4_is_the_documented_permutation(E, I, H):
    G.say(f"case: MXFP4 pack E={E} I={I} H={H}")
    g = torch.Generator(device="cuda")
    g.manual_seed(E * 7919 + I)
    rnd = lambda *shape: torch.randint(0, 256, shape, generator=g, device="cuda", dtype=torch.int32).to(torch.uint8)
    w1, w3 = (rnd(E, I, H // 2), rnd(E, I, H // 32)), (rnd(E, I, H // 2), rnd(E, I, H // 32))
    w2 = (rnd(E, H, I // 2), rnd(E, H, I // 32))
    (uc, us), (dc, ds) = B.pack_mxfp4_expert_weights(w1, w3, w2)
    torch.cuda.synchronize()
    h = lambda t: t.cpu().numpy()
    # up codes: per (expert, 16-row wave band, slot of 2 k-steps), lane = 16 g + r holds the
    # dwords (W1 step 0, W1 step 1, W3 step 0, W3 step 1) of row r, k-group g; the wave
    # bands of a workgroup band (4 of them) lie side by side slot by slot
    ns = H // 64
    parts = [_dwords(h(c)).reshape(E, I // 16, 16, ns, 2, 4) for c in (w1[0], w3[0])]
    ref = np.stack([p.transpose(0, 1, 3, 5, 2, 4) for p in parts], axis=-2)  # [E,nb,ns,g,r,m,j]
    assert np.array_equal(_dwords(h(uc)), _wg_bands(ref))
    parts = [h(s).reshape(E, I // 16, 16, ns, 2) for s in (w1[1], w3[1])]
    ref = np.stack([p.transpose(0, 1, 3, 2, 4) for p in parts], axis=-2)       # [E,nb,ns,r,m,j]
    assert np.array_equal(h(us), _wg_bands(ref))
    # down: the two 16-row halves of each 32-row band of W2
    ns = I // 64
    p = _dwords(h(w2[0])).reshape(E, H // 32, 2, 16, ns, 2, 4)
    ref = p.transpose(0, 1, 4, 6, 3, 2, 5)                                      # [E,nb,ns,g,r,m,j]
    assert np.array_equal(_dwords(h(dc)), _wg_bands(ref))
    p = h(w2[1]).reshape(E, H // 32, 2, 16, ns, 2)
    assert np.array_equal(h(ds), _wg_bands(p.transpose(0, 1, 4, 3, 2, 5)))


# ---------------------------------------------------------------------------- FFN parity

@pytest.mark.parametrize("E,K,H,I,T", [
    (8, 2, 192, 320, 8),      # one token tile; up: a lone tail chunk, down: a partial row band
    (8, 2, 192, 320, 24),     # the two-tile kernel; buckets of about 6 take its one-tile pass
    (6, 3, 256, 128, 100),    # buckets of about 50 tokens: four token tiles
    (4, 2, 256, 128, 200),    # buckets of about 100 tokens: two token groups
    (256, 4, 128, 128, 100),  # the most experts: the union fills four positions a lane
    (4, 2, 2880, 2880, 40),   # full-size reductions: 11 whole chunks and a tail
])
def test_mxfp4_layer_matches_oracle(E, K, H, I, T):
    G.say(f"case: MXFP4 layer E={E} top-{K} H={H} I={I} T={T}, gate-routed")
    layer = MxLayer(synth.LayerShape("mx", E=E, K=K, H=H, I=I), T, seed=E + T)
    _check_layer(layer, layer.run())


@pytest.mark.parametrize("T,heavy", [(24, [(2, 24), (5, 17)]),
                                     (32, [(3, 17), (7, 24), (11, 32)])])
def test_mxfp4_two_tile_pass(T, heavy):
    # 16 < T <= 32 takes the two-tile kernel; buckets of 17, 24 and 32 tokens
    # run its two-tile pass.  H = 640 is two full 8-step chunks and a tail.
    sh = synth.LayerShape("mx_two_tile", E=16, K=4, H=640, I=320)
    G.say(f"case: MXFP4 E=16 top-4 H=640 I=320 T={T}, buckets of {[n for _, n in heavy]} tokens")
    ids, w = G.fixed_bucket_routing(T, sh.E, sh.K, heavy, seed=T + 1)
    layer = MxLayer(sh, T, seed=T)
    g = layer.run((ids, w))
    assert [int(g["counts"][e]) for e, _ in heavy] == [n for _, n in heavy]
    _check_layer(layer, g, (ids.astype(np.int64), w))


def test_mxfp4_full_code_and_scale_range():
    # random codes over all 16 E2M1 values (signed zeros, subnormal 0.5, +-6) and
    # scale codes spread over 41 binades, on every expert
    G.say("case: MXFP4 random codes, scale codes 100..140, E=6 top-2 H=128 I=192 T=20")
    sh = synth.LayerShape("mx_range", E=6, K=2, H=128, I=192)
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    rnd = lambda lo, hi, *shape: torch.randint(lo, hi, shape, generator=g, device="cuda",
                                               dtype=torch.int32).to(torch.uint8)
    q = {"w1": (rnd(0, 256, 6, 192, 64), rnd(100, 141, 6, 192, 4)),
         "w3": (rnd(0, 256, 6, 192, 64), rnd(100, 141, 6, 192, 4)),
         "w2": (rnd(0, 256, 6, 128, 96), rnd(100, 141, 6, 128, 6))}
    layer = MxLayer(sh, 20, seed=5, q=q)
    ids, w, _ = synth.controlled_routing(20, 6, 2, U=6, seed=5)
    g = layer.run((ids, w))
    G.compare_buckets(g, ids, sh.E)
    qh = layer.host_q()
    b = O.bucket(ids, sh.E)
    with np.errstate(over="ignore"):
        y = MX.expert_ffn(layer.x_np, qh["w1"], qh["w3"], qh["w2"], ids, b)
    # outputs reach 1e14 here, so the absolute MAE bar is replaced by its
    # scale-free form (MAE relative to the mean output magnitude)
    nw, mae = G.output_errors(g["y_slots"], y)
    rel_mae = mae / np.abs(y).mean()
    G.say(f"  normwise max rel err {nw:.3e}, MAE / mean|ref| {rel_mae:.3e}")
    assert nw <= G.OUT_NORMWISE_DESIGN and rel_mae <= G.OUT_MAE


def test_mxfp4_equals_bf16_path_on_dequantized_weights():
    G.say("case: MXFP4 vs bf16 path on the dequantized weights, E=6 top-3 H=256 I=128 T=100")
    sh = synth.LayerShape("mx_eq", E=6, K=3, H=256, I=128)
    layer = MxLayer(sh, 100, seed=3)
    g = layer.run()
    q = layer.host_q()
    bf = []
    for name in ("w1", "w3", "w2"):
        wf = MX.dequantize(*q[name]).astype(np.float32)     # exact: every value is a bf16 number
        assert not (wf.view(np.uint32) & 0xFFFF).any()
        bf.append(torch.from_numpy(wf).cuda().to(torch.bfloat16))
    p13, p2 = B.pack_expert_weights(*bf)
    buf = B.LayerBuffers.allocate(layer.d)
    B.moe_layer(layer.x, layer.wg, p13, p2, layer.d, buf)
    torch.cuda.synchronize()
    r = G.fetch(buf, layer.d)
    assert np.array_equal(r["ids"], g["ids"])
    assert np.array_equal(r["y_slots"], g["y_slots"]), "MXFP4 and bf16 paths differ"
    assert np.array_equal(r["out"], g["out"])


def test_mxfp4_big_buckets_take_token_groups():
    G.say("case: MXFP4 320 tokens on 8 of 16 experts (buckets of ~80), H=256 I=192")
    sh = synth.LayerShape("mx_big", E=16, K=2, H=256, I=192)
    layer = MxLayer(sh, 320, seed=8)
    ids, w, _ = synth.controlled_routing(320, 16, 2, U=8, seed=8)
    g = layer.run((ids, w))
    G.say(f"  max bucket {g['counts'].max()}")
    assert g["counts"].max() > 64
    _check_layer(layer, g, (ids, w))


@pytest.mark.parametrize("n", [32, 33, 64, 65])
def test_mxfp4_large_batch_dealing_boundary(n):
    # Batches over 64 tokens deal whole experts while every bucket fits one
    # 32-token MXFP4 group, and (expert, band) units once one does not (33:
    # two groups; 64/65: two and three).
    sh = synth.LayerShape("mx_dealing", E=16, K=4, H=256, I=192)
    T = 80
    G.say(f"case: MXFP4 E=16 top-4 H=256 I=192 T={T}, expert 5 takes {n} tokens")
    ids, w = G.fixed_bucket_routing(T, sh.E, sh.K, [(5, n)], seed=n)
    layer = MxLayer(sh, T, seed=n)
    g = layer.run((ids, w))
    assert int(g["counts"][5]) == n and int(g["counts"].max()) == n
    _check_layer(layer, g, routing=(ids, w))


@pytest.mark.parametrize("H,I,T", [(B.MOE_MAX_H, 256, 24), (256, B.MOE_MAX_I, 80)])
def test_mxfp4_largest_hidden_and_intermediate(H, I, T):
    # The limits on H and I with MXFP4 experts: 256 ring slots a reduction.
    sh = synth.LayerShape("mx_max_hi", E=4, K=2, H=H, I=I)
    G.say(f"case: MXFP4 E=4 top-2 H={H} I={I} T={T}, expert 1 takes every token")
    ids, w = G.fixed_bucket_routing(T, sh.E, sh.K, [(1, T)], seed=T)
    layer = MxLayer(sh, T, seed=(H + I) % 1000)
    g = layer.run((ids, w))
    assert int(g["counts"][1]) == T
    _check_layer(layer, g, routing=(ids, w))


@pytest.mark.parametrize("path", B.FFN_PATHS)
def test_mxfp4_layer_output_does_not_depend_on_the_batch(path):
    """As for bf16 experts: a token's layer output is the same bits in any batch,
    on both sides of the 64-token kernel switch and of the 32-token group."""
    sh = synth.LayerShape("mx_batch", E=32, K=4, H=512, I=384)
    G.say(f"case: MXFP4 E=32 top-4 H=512 I=384, 256-token batch vs sub-batches, path {path}")
    layer = MxLayer(sh, 256, seed=24)
    d = layer.d
    B.moe_layer_mxfp4(layer.x, layer.wg, layer.up, layer.down, d, layer.buf, path=path)
    torch.cuda.synchronize()
    full = G.fetch(layer.buf, d)
    for t0, t1 in [(0, 1), (0, 16), (16, 80), (100, 164), (0, 65), (80, 209), (3, 256)]:
        ds = B.dims(t1 - t0, sh.H, sh.E, sh.K, sh.I)
        buf = B.LayerBuffers.allocate(ds)
        B.moe_layer_mxfp4(layer.x[t0:t1].contiguous(), layer.wg, layer.up, layer.down, ds, buf,
                          path=path)
        torch.cuda.synchronize()
        part = G.fetch(buf, ds)
        for k in ("ids", "weights", "out"):
            assert np.array_equal(full[k][t0:t1], part[k]), f"{k} of tokens {t0}..{t1 - 1} differ"


def test_mxfp4_empty_batch_and_invalid_routing():
    G.say("case: MXFP4 empty batch, then a duplicated id (invalid routing)")
    sh = synth.LayerShape("mx_edge", E=8, K=2, H=128, I=64)
    layer = MxLayer(sh, 6, seed=2)
    d0 = B.dims(0, sh.H, sh.E, sh.K, sh.I)
    B.moe_expert_ffn_mxfp4(layer.x, layer.up, layer.down, layer.buf.offsets, layer.buf.perm_token,
                           layer.buf.union_ids, layer.buf.union_size, d0, layer.buf.y_perm,
                           layer.buf.ws)
    ids = np.array([[0, 1], [2, 2], [3, 4], [5, 6], [7, 0], [1, 2]], np.int32)  # token 1 repeats 2
    w = np.full((6, 2), 0.5, np.float32)
    layer.buf.y_perm.fill_(123.0)
    g = layer.run((ids, w))
    assert g["union_size"] == -1
    assert np.all(g["y_slots"] == 123.0), "the FFN wrote outputs for invalid routing"


# ---------------------------------------------------------------------------- full gpt-oss shape

@pytest.fixture(scope="module")
def gpt_oss_mx():
    G.say("building the gpt-oss-shaped MXFP4 layer (E=128 top-4 H=I=2880), T=256")
    return MxLayer(GPTOSS, 256)


def _every_row(layer: MxLayer, g: dict, ids, wts, label):
    """Every slot row and every output row against the oracle on the given
    routing (the oracle dequantizes each union expert's matrices once)."""
    ids = np.asarray(ids, np.int64)
    q = layer.host_q(sorted(set(ids.ravel().tolist())))
    ref = MX.moe_layer_routed(layer.x_np, ids, np.asarray(wts, np.float64), q["w1"], q["w3"],
                              q["w2"], GPTOSS.E)
    G.check_output(g["y_slots"], ref["y_slots"], f"every slot, {label}")
    G.check_output(g["out"], ref["out"], f"every token, {label}")


def test_gpt_oss_mxfp4_gate_routed(gpt_oss_mx):
    G.say("case: gpt-oss MXFP4 layer T=256, gate-routed, all tokens and slots")
    g = gpt_oss_mx.run()
    G.say(f"  union size {g['union_size']}, max bucket {g['counts'].max()}")
    near = G.check_gate(g, gpt_oss_mx.x_np, gpt_oss_mx.wg_np, GPTOSS.K)
    ids = g["ids"].astype(np.int64)
    G.compare_buckets(g, ids, GPTOSS.E)
    # on the GPU's own routing, whose near-tie picks check_gate has validated
    _every_row(gpt_oss_mx, g, ids, g["weights"], f"gate-routed ({int(near.sum())} near-ties)")


@pytest.mark.parametrize("U", [32, 128])
def test_gpt_oss_mxfp4_controlled_union(gpt_oss_mx, U):
    G.say(f"case: gpt-oss MXFP4 layer T=256, controlled union U={U}, all tokens and slots")
    ids, w, _ = synth.controlled_routing(256, GPTOSS.E, GPTOSS.K, U=U, seed=U)
    g = gpt_oss_mx.run((ids, w))
    G.compare_buckets(g, ids, GPTOSS.E)
    G.say(f"  union size {g['union_size']}, max bucket {g['counts'].max()}")
    _every_row(gpt_oss_mx, g, ids, w, f"U={U}")
