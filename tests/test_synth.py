"""Seeded input generators: shapes, determinism and the statistics each workload promises."""
import numpy as np
import pytest
import torch

from paper_2607_00466_amd import synth


def test_shapes_and_dtypes():
    s = synth.SHAPES["tiny"]
    x = synth.hidden_states(8, s.H)
    wg = synth.gate_weights(s)
    w1, w3, w2 = synth.expert_weights(s)
    assert x.shape == (8, 256) and x.dtype == np.float32
    assert wg.shape == (16, 256) and wg.dtype == np.float32
    assert w1.shape == (16, 128, 256) and w3.shape == (16, 128, 256) and w2.shape == (16, 256, 128)
    assert w1.dtype == torch.bfloat16
    assert synth.bf16_bits(w1).dtype == np.uint16
    assert s.expert_bytes == 196608
    assert synth.SHAPES["qwen3_30b_a3b"].expert_bytes == 9437184
    assert synth.SHAPES["gpt_oss_120b"].expert_bytes == 49766400


def test_deterministic_and_distinct_streams():
    s = synth.SHAPES["tiny"]
    assert np.array_equal(synth.hidden_states(4, 64, seed=3), synth.hidden_states(4, 64, seed=3))
    assert not np.array_equal(synth.hidden_states(4, 64, seed=3), synth.hidden_states(4, 64, seed=4))
    a = synth.bf16_bits(synth.expert_weights(s, seed=1)[0])
    b = synth.bf16_bits(synth.expert_weights(s, seed=1)[0])
    assert np.array_equal(a, b)
    assert not np.array_equal(a, synth.bf16_bits(synth.expert_weights(s, seed=1, layer=1)[0]))


def test_weight_statistics():
    s = synth.SHAPES["tiny"]
    w = synth.expert_weights(s)[0].float().numpy()
    assert abs(w.std() - 0.02) < 5e-4 and abs(w.mean()) < 5e-4
    g = synth.gate_weights(s)
    assert abs(g.std() - 0.02) < 1e-3


@pytest.mark.parametrize("U", [8, 16, 32, 64, 96, 128])
def test_controlled_routing(U):
    T, E, K = 64, 128, 8
    ids, w, subset = synth.controlled_routing(T, E, K, U, seed=0)
    assert ids.shape == (T, K) and ids.dtype == np.int32
    assert len(set(subset.tolist())) == U
    for row in ids:
        assert len(set(row.tolist())) == K
        assert set(row.tolist()) <= set(subset.tolist())
    np.testing.assert_allclose(w.sum(1), 1.0, atol=1e-6)
    assert np.all(w > 0)


def test_controlled_union_expectation():
    # Realised union over many batches vs the closed form U (1 - (1 - K/U)^T).
    T, E, K, U = 8, 128, 8, 32
    sizes = [len(set(synth.controlled_routing(T, E, K, U, seed=s)[0].ravel().tolist())) for s in range(300)]
    expect = U * (1 - (1 - K / U) ** T)
    assert abs(np.mean(sizes) - expect) < 0.35


def test_domain_routing():
    m = synth.DomainModel()
    L = 3
    subs = synth.domain_subsets(m, L, seed=0)
    assert subs.shape == (8, L, 32)
    batches = synth.domain_batches(m, 128)
    assert set(batches) == {f"same_{d}" for d in range(8)} | {"mixed"}
    assert np.bincount(batches["mixed"]).tolist() == [16] * 8
    ids, w = synth.domain_routing(m, subs, batches["same_0"], layer=0, seed=0)
    assert ids.shape == (128, 8)
    for row in ids:
        assert len(set(row.tolist())) == 8
    np.testing.assert_allclose(w.sum(1), 1.0, atol=1e-6)
    # about 80% of picks come from the domain subset (plus uniform picks that land in it)
    inside = np.isin(ids, subs[0, 0]).mean()
    assert 0.78 < inside < 0.92
    # a same-domain batch activates fewer distinct experts than a mixed one
    same = np.mean([len(set(synth.domain_routing(m, subs, batches[f"same_{d}"], 0)[0].ravel().tolist()))
                    for d in range(8)])
    mixed = len(set(synth.domain_routing(m, subs, batches["mixed"], 0)[0].ravel().tolist()))
    assert same < mixed


def test_mxfp4_weights_shapes_and_determinism():
    sh = synth.SHAPES["tiny"]
    a = synth.mxfp4_expert_weights(sh, seed=3, experts=2)
    b = synth.mxfp4_expert_weights(sh, seed=3, experts=2)
    for name, (rows, cols) in (("w1", (sh.I, sh.H)), ("w3", (sh.I, sh.H)), ("w2", (sh.H, sh.I))):
        c, s = a[name]
        assert c.dtype == torch.uint8 and s.dtype == torch.uint8
        assert tuple(c.shape) == (2, rows, cols // 2) and tuple(s.shape) == (2, rows, cols // 32)
        assert torch.equal(c, b[name][0]) and torch.equal(s, b[name][1])
        assert 1 <= int(s.min()) and int(s.max()) <= 252
    # the same fp32 draws as the bf16 weights: both round the same numbers
    w1 = synth.expert_weights(sh, seed=3, experts=2)[0].float()
    c, s = a["w1"]
    X = torch.pow(2.0, s.float() - 127).repeat_interleave(32, dim=-1)
    assert (w1.abs() <= 8 * X).all()
