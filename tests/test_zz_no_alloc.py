"""moe_expert_ffn_noalloc (the library's fixed per-GPU workspace) against
moe_expert_ffn (a caller workspace), bit for bit, on two calls in a row, the
second with a smaller problem, through the C ABI."""
import numpy as np
import pytest
import torch

from paper_2607_00466_amd import binding as B
from paper_2607_00466_amd import synth
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

QWEN = synth.SHAPES["qwen3_30b_a3b"]


def _compare(shape, T, U, seed):
    G.say(f"case: noalloc vs workspace FFN, E={shape.E} top-{shape.K} H={shape.H} I={shape.I} "
          f"T={T} controlled U={U}")
    layer = G.Layer(shape, T, seed=seed, experts_on_host=False)
    d, buf = layer.d, layer.buf
    ids, _, _ = synth.controlled_routing(T, shape.E, shape.K, U, seed=seed)
    B.moe_bucket(torch.from_numpy(ids).cuda(), d, buf.counts, buf.offsets, buf.perm_token,
                 buf.pair_pos, buf.union_ids, buf.union_size)
    ref = torch.full_like(buf.y_perm, float("nan"))
    got = torch.full_like(buf.y_perm, float("nan"))
    B.moe_expert_ffn(layer.x, layer.p13, layer.p2, buf.offsets, buf.perm_token, buf.union_ids,
                     buf.union_size, d, ref, buf.ws)
    B.moe_expert_ffn_noalloc(layer.x, layer.p13, layer.p2, buf.offsets, buf.perm_token,
                             buf.union_ids, buf.union_size, d, got)
    torch.cuda.synchronize()
    P = T * shape.K
    assert not torch.isnan(ref[:P]).any(), "the workspace call left slots unwritten"
    assert torch.equal(got[:P], ref[:P]), "noalloc and workspace FFN differ"
    G.say(f"  equal on all {P} slots; workspace {B.moe_ffn_workspace_bytes(d)} bytes "
          f"of {B.load().moe_expert_ffn_noalloc_max_bytes()}")


def test_noalloc_ffn_matches_workspace_ffn_twice():
    # the first call fills more of the fixed workspace than the second reads
    _compare(QWEN, 64, 32, seed=21)
    _compare(QWEN, 16, 16, seed=22)


def test_noalloc_ffn_rejects_oversize():
    d = B.dims(2048, QWEN.H, QWEN.E, 16, QWEN.I)  # 100 MB of workspace
    x = torch.zeros((d.T, d.H), device="cuda")
    w13 = torch.zeros(2 * d.E * d.I * d.H, dtype=torch.bfloat16, device="cuda")
    w2 = torch.zeros(d.E * d.H * d.I, dtype=torch.bfloat16, device="cuda")
    buf = B.LayerBuffers.allocate(d)
    with pytest.raises(B.MoeError) as err:
        B.moe_expert_ffn_noalloc(x, w13, w2, buf.offsets, buf.perm_token, buf.union_ids,
                                 buf.union_size, d, buf.y_perm)
    assert err.value.status == B.MOE_ERR_WORKSPACE
