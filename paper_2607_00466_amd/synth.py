"""Seeded synthetic inputs for the batched-decode MoE layer.

This module only draws random numbers and lays them out; it holds none of the
layer's arithmetic (no gate, no selection, no bucketing, no FFN, no combine).
Both the HIP path and the CPU oracle consume what it produces, so the two never
disagree about an input.

The paper measures the layer on real models with public datasets (Evaluation,
"Models" and "Datasets"); none of that is available here, so every workload is
synthetic with the model's shape:

* ``tiny``            E=16,  top-2, hidden 256,  expert intermediate 128
* ``qwen3_30b_a3b``   E=128, top-8, hidden 2048, expert intermediate 768
* ``gpt_oss_120b``    E=128, top-4, hidden 2880, expert intermediate 2880

E and top-k per model are those the paper lists (Evaluation, "Models"); hidden
and intermediate sizes are the public model shapes.  Weights are
N(0, 0.02) drawn in fp32 and rounded to bf16 (round-to-nearest-even, which is
what ``torch.Tensor.to(torch.bfloat16)`` does); the gate stays fp32; hidden
states are N(0, 1) fp32.

Storage layout (row-major, "[out, in]" so each output neuron's weights are
contiguous along the reduction axis):

* gate  ``w_gate`` [E, H]  fp32
* W1 (SwiGLU gate proj) ``w1`` [E, I, H] bf16
* W3 (SwiGLU up proj)   ``w3`` [E, I, H] bf16
* W2 (down proj)        ``w2`` [E, H, I] bf16

Routing generators (used when the gate is bypassed) return ``ids`` [T, K]
int32 (distinct within a token) and ``weights`` [T, K] fp32 summing to one per
token.  ``prefill_picks`` draws the picks of a prefill forward over many MoE
layers, for the expert-signature cache.

``mxfp4_expert_weights`` gives the same draws quantized to MXFP4 (the format
the paper serves GPT-OSS-120B in, Evaluation "Models"), per the OCP
Microscaling specification: FP4 E2M1 codes, two a byte with the lower index in
the low nibble, [E, R, K/2] uint8, and one E8M0 scale per 32 values along the
reduction axis, [E, R, K/32] uint8.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

WEIGHT_STD = 0.02

# Fixed child indices of SeedSequence(seed).spawn(...) so that each kind of
# draw has its own stream, stable when other draws are added or resized.
_STREAM_X = 0
_STREAM_GATE = 1
_STREAM_EXPERTS = 2
_STREAM_ROUTING = 3
_STREAM_PREFILL = 4
_STREAM_REQUESTS = 5
_N_STREAMS = 8


@dataclass(frozen=True)
class LayerShape:
    """Shape of one MoE layer: E experts, top-K, hidden H, expert intermediate I."""

    name: str
    E: int
    K: int
    H: int
    I: int

    @property
    def expert_bytes(self) -> int:
        """bf16 bytes of one expert's W1, W3 and W2."""
        return 3 * self.H * self.I * 2


SHAPES = {
    "tiny": LayerShape("tiny", E=16, K=2, H=256, I=128),
    "qwen3_30b_a3b": LayerShape("qwen3_30b_a3b", E=128, K=8, H=2048, I=768),
    "gpt_oss_120b": LayerShape("gpt_oss_120b", E=128, K=4, H=2880, I=2880),
}


def _streams(seed: int) -> list[np.random.SeedSequence]:
    return np.random.SeedSequence(seed).spawn(_N_STREAMS)


def _rng(seed: int, stream: int, *extra: int) -> np.random.Generator:
    ss = _streams(seed)[stream]
    if extra:
        ss = np.random.SeedSequence(ss.generate_state(4).tolist() + list(extra))
    return np.random.default_rng(ss)


def _torch_seed(seed: int, stream: int, *extra: int) -> int:
    ss = _streams(seed)[stream]
    state = np.random.SeedSequence(ss.generate_state(4).tolist() + list(extra)).generate_state(2, np.uint64)
    return int(state[0] & np.uint64((1 << 63) - 1))


def hidden_states(T: int, H: int, seed: int = 0, layer: int = 0) -> np.ndarray:
    """Decode-batch hidden states x [T, H] fp32, N(0, 1)."""
    return _rng(seed, _STREAM_X, layer).standard_normal((T, H), dtype=np.float32)


def gate_weights(shape: LayerShape, seed: int = 0, layer: int = 0) -> np.ndarray:
    """Gate weights stored [E, H] fp32, N(0, 0.02)."""
    g = _rng(seed, _STREAM_GATE, layer).standard_normal((shape.E, shape.H), dtype=np.float32)
    return (g * np.float32(WEIGHT_STD)).astype(np.float32)


def expert_weights(shape: LayerShape, seed: int = 0, layer: int = 0, device: str = "cpu",
                   experts: int | None = None) -> tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Expert weights (w1 [E,I,H], w3 [E,I,H], w2 [E,H,I]) as torch bf16 tensors.

    Drawn with a seeded torch generator on ``device`` (fp32 N(0, 0.02), then
    round-to-nearest-even to bf16), one expert at a time to bound the fp32
    temporary.  The same (seed, layer, device) always yields the same bits.
    ``experts`` limits E (used by tests that need only the first few experts).
    """
    E = shape.E if experts is None else experts
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(_torch_seed(seed, _STREAM_EXPERTS, layer))
    out = []
    for rows, cols in ((shape.I, shape.H), (shape.I, shape.H), (shape.H, shape.I)):
        w = torch.empty((E, rows, cols), dtype=torch.bfloat16, device=dev)
        for e in range(E):
            tmp = torch.randn((rows, cols), generator=gen, dtype=torch.float32, device=dev)
            w[e].copy_(tmp.mul_(WEIGHT_STD))
        out.append(w)
    return out[0], out[1], out[2]


def _mxfp4_quantize(w: torch.Tensor) -> tuple[torch.Tensor, torch.Tensor]:
    """fp32 [R, K] -> MXFP4 (codes uint8 [R, K/2], scales uint8 [R, K/32]).

    The conversion of the OCP Microscaling specification: per block of 32
    consecutive values, shared exponent floor(log2(max |v|)) - 2 (2 is the
    largest exponent of FP4 E2M1), stored as the E8M0 code exponent + 127;
    each v / 2^exponent is rounded to the nearest E2M1 magnitude
    {0, 0.5, 1, 1.5, 2, 3, 4, 6} (ties to the even code), saturating at 6.
    Two codes a byte, the lower index in the low nibble.  This only makes
    inputs: the layer's arithmetic (dequantization included) is elsewhere.
    """
    R, K = w.shape
    v = w.reshape(R, K // 32, 32)
    amax = v.abs().amax(dim=-1)
    _, ex = torch.frexp(amax)                       # amax = m * 2^ex, m in [0.5, 1)
    shared = (ex - 1 - 2).clamp(-126, 125)          # codes 1 .. 252
    scaled = torch.ldexp(v, (-shared).unsqueeze(-1).to(v.dtype))
    mag = scaled.abs()
    # index into the E2M1 magnitudes; at a midpoint '>' keeps the lower (even)
    # code and '>=' takes the upper (even) one
    idx = ((mag > 0.25).to(torch.uint8) + (mag >= 0.75) + (mag > 1.25) + (mag >= 1.75)
           + (mag > 2.5) + (mag >= 3.5) + (mag > 5.0))
    sign = ((scaled < 0) & (idx > 0)).to(torch.uint8) << 3
    nib = (idx | sign).reshape(R, K)
    codes = nib[:, 0::2] | (nib[:, 1::2] << 4)
    scales = (shared + 127).to(torch.uint8)
    return codes.contiguous(), scales.contiguous()


def mxfp4_expert_weights(shape: LayerShape, seed: int = 0, layer: int = 0, device: str = "cpu",
                         experts: int | None = None) -> dict[str, tuple[torch.Tensor, torch.Tensor]]:
    """MXFP4 expert weights {"w1", "w3", "w2": (codes, scales)} as torch uint8.

    The fp32 N(0, 0.02) draws are those of ``expert_weights`` (same generator,
    seed and order), quantized per OCP MX instead of rounded to bf16: codes
    [E, R, K/2] and scales [E, R, K/32], blocks along the reduction axis.
    """
    E = shape.E if experts is None else experts
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(_torch_seed(seed, _STREAM_EXPERTS, layer))
    out = {}
    for name, (rows, cols) in (("w1", (shape.I, shape.H)), ("w3", (shape.I, shape.H)),
                               ("w2", (shape.H, shape.I))):
        codes = torch.empty((E, rows, cols // 2), dtype=torch.uint8, device=dev)
        scales = torch.empty((E, rows, cols // 32), dtype=torch.uint8, device=dev)
        for e in range(E):
            tmp = torch.randn((rows, cols), generator=gen, dtype=torch.float32, device=dev)
            c, s = _mxfp4_quantize(tmp.mul_(WEIGHT_STD))
            codes[e].copy_(c)
            scales[e].copy_(s)
        out[name] = (codes, scales)
    return out


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Host copy of a bf16 tensor as raw uint16 bit patterns."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def dirichlet_weights(T: int, K: int, rng: np.random.Generator) -> np.ndarray:
    """Routing weights [T, K] fp32 ~ Dirichlet(1, ..., 1) per token."""
    return rng.dirichlet(np.ones(K), size=T).astype(np.float32)


def controlled_routing(T: int, E: int, K: int, U: int, seed: int = 0, layer: int = 0
                       ) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Gate-bypassed routing with a controlled expert union.

    A fixed random subset of U experts is drawn once; each token then picks K
    distinct ids uniformly from that subset, with Dirichlet(1) weights.
    Returns (ids [T,K] int32, weights [T,K] fp32, subset [U] int32).
    """
    if not (1 <= K <= U <= E):
        raise ValueError(f"need 1 <= K <= U <= E, got K={K} U={U} E={E}")
    rng = _rng(seed, _STREAM_ROUTING, layer, U, T)
    subset = rng.choice(E, size=U, replace=False).astype(np.int32)
    ids = np.empty((T, K), dtype=np.int32)
    for t in range(T):
        ids[t] = subset[rng.choice(U, size=K, replace=False)]
    return ids, dirichlet_weights(T, K, rng), subset


@dataclass(frozen=True)
class DomainModel:
    """Domain-clustered routing: per (domain, layer) an ordered preferred subset."""

    E: int = 128
    K: int = 8
    n_domains: int = 8
    subset_size: int = 32
    p_domain: float = 0.8
    zipf_s: float = 1.1


def domain_subsets(model: DomainModel, n_layers: int, seed: int = 0) -> np.ndarray:
    """Preferred subsets [n_domains, n_layers, subset_size] int32 (ordered by Zipf rank)."""
    rng = _rng(seed, _STREAM_ROUTING, 0x0D0)
    out = np.empty((model.n_domains, n_layers, model.subset_size), dtype=np.int32)
    for d in range(model.n_domains):
        for layer in range(n_layers):
            out[d, layer] = rng.choice(model.E, size=model.subset_size, replace=False)
    return out


def domain_routing(model: DomainModel, subsets: np.ndarray, token_domains: np.ndarray,
                   layer: int, seed: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """One layer's routing for tokens with the given domains.

    Each of a token's K picks is, with probability p_domain, the rank-r expert
    of its domain's subset with r ~ truncated Zipf(s) over 1..subset_size, and
    otherwise uniform over all E experts; a pick equal to one already made for
    that token is drawn again.  Weights are Dirichlet(1).
    """
    T = int(token_domains.shape[0])
    rng = _rng(seed, _STREAM_ROUTING, 0x0D1, layer, T, int(token_domains.sum()))
    ranks = np.arange(1, model.subset_size + 1, dtype=np.float64)
    pz = ranks ** (-model.zipf_s)
    pz /= pz.sum()
    ids = np.empty((T, model.K), dtype=np.int32)
    for t in range(T):
        sub = subsets[token_domains[t], layer]
        chosen: list[int] = []
        while len(chosen) < model.K:
            if rng.random() < model.p_domain:
                e = int(sub[rng.choice(model.subset_size, p=pz)])
            else:
                e = int(rng.integers(model.E))
            if e not in chosen:
                chosen.append(e)
        ids[t] = chosen
    return ids, dirichlet_weights(T, model.K, rng)


def domain_batches(model: DomainModel, T: int, seed: int = 0) -> dict[str, np.ndarray]:
    """Token-domain assignments for a same-domain batch per domain and an even mix."""
    if T % model.n_domains:
        raise ValueError("T must be a multiple of the number of domains for the mixed batch")
    out = {f"same_{d}": np.full(T, d, dtype=np.int64) for d in range(model.n_domains)}
    out["mixed"] = np.repeat(np.arange(model.n_domains, dtype=np.int64), T // model.n_domains)
    return out


def prefill_picks(n_layers: int, T: int, E: int, K: int, seed: int = 0, skew: float = 0.0
                  ) -> np.ndarray:
    """Top-k picks of T prefill tokens at n_layers MoE layers, int32 [n_layers, T, K].

    Each token's K picks at a layer are distinct.  skew = 0 draws them
    uniformly; skew > 0 draws them from a Zipf(skew) popularity over a random
    permutation of the experts per layer (a few experts are hot).
    """
    rng = _rng(seed, _STREAM_PREFILL, n_layers, T, E, K)
    out = np.empty((n_layers, T, K), dtype=np.int32)
    for layer in range(n_layers):
        if skew > 0:
            order = rng.permutation(E)
            p = np.arange(1, E + 1, dtype=np.float64) ** (-skew)
            p /= p.sum()
        for t in range(T):
            if skew > 0:
                out[layer, t] = order[rng.choice(E, size=K, replace=False, p=p)]
            else:
                out[layer, t] = rng.choice(E, size=K, replace=False)
    return out


def domain_pick_probs(model: DomainModel, subsets: np.ndarray, domain: int, layer: int) -> np.ndarray:
    """Per-expert pick propensities of one domain at one layer, float64 [E]:
    p_domain times the truncated Zipf(s) weight of the expert's rank in the
    domain's subset, plus (1 - p_domain) / E for every expert."""
    ranks = np.arange(1, model.subset_size + 1, dtype=np.float64)
    pz = ranks ** (-model.zipf_s)
    pz /= pz.sum()
    p = np.full(model.E, (1.0 - model.p_domain) / model.E)
    p[subsets[domain, layer]] += model.p_domain * pz
    return p


def domain_requests(model: DomainModel, subsets: np.ndarray, domains: np.ndarray, n_tokens: int,
                    seed: int = 0, stream: int = 0) -> np.ndarray:
    """Top-k picks of n_tokens tokens of each request, at every layer:
    int32 [n_layers, n_requests, n_tokens, K].

    A token of a request with domain d takes its K distinct picks at layer l
    by successive draws from domain_pick_probs(d, l), each draw excluding the
    experts already picked (Gumbel-top-K over log-propensities, which is that
    successive sampling).  Vectorised; `stream` separates independent draws
    (for example a request's prefill and its decode steps).
    """
    n_layers = subsets.shape[1]
    R = len(domains)
    rng = _rng(seed, _STREAM_REQUESTS, stream, R, n_tokens, n_layers)
    out = np.empty((n_layers, R, n_tokens, model.K), dtype=np.int32)
    for layer in range(n_layers):
        logp = np.log(np.stack([domain_pick_probs(model, subsets, d, layer)
                                for d in range(model.n_domains)]))
        keys = logp[domains][:, None, :] + rng.gumbel(size=(R, n_tokens, model.E))
        top = np.argpartition(-keys, model.K - 1, axis=2)[:, :, :model.K]
        out[layer] = top.astype(np.int32)
    return out
