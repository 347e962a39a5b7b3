"""Benchmark of the batched-decode MoE layer on one MI355X.

Default workload: one Qwen3-30B-A3B-shaped MoE layer (E=128 experts, top-8,
hidden 2048, expert intermediate 768, SwiGLU, bf16 experts, fp32 gate), a
decode batch of 64 tokens routed by the gate.  A step is one whole layer:
gate scores and top-k, buckets and union, expert FFNs (up and down), combine.
Inputs are synthetic and resident in HBM before the timed region.

To keep the 256 MB Infinity Cache from serving repeated weight reads, step i
uses weight copy i mod R, with R copies whose union bytes together exceed
2 GB (all copies hold the same bits).

The timed layer steps are HIP graph replays, each graph holding several
consecutive layer steps (as a captured decode step holds its layers), so host
launch cost is not in the GPU timeline.  Printed: one JSON line with the layer's achieved algorithmic GB/s
(the metric), the roofline of the dominant kernel (the FFN up projection,
timed with HIP events on the stream it runs on), the CPU oracle's rate on
the host cores, and the controlled-union and batch sweeps of the paper's
motivating measurement with a least-squares fit of latency against the union
(``--no-sweep`` leaves them out; ``--sweep PATH`` also writes them to PATH as
JSON lines; ``--point T:U`` times single controlled points only).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2607_00466_amd import binding as B  # noqa: E402
from paper_2607_00466_amd import synth  # noqa: E402

METRIC = "MoE decode-layer µs and achieved HBM GB/s vs distinct-expert union (Qwen3-30B-A3B shape)"
HBM_PEAK_GBS = 8000.0
ROTATE_BYTES = 2 << 30
LAYERS_PER_GRAPH = 8
# How each layer step runs the expert FFN (binding.FFN_PATHS): "routed" is
# moe_expert_ffn_up_routed then moe_expert_ffn_down (measured faster than the
# one-launch moe_expert_ffn_routed at every union size).
FFN_PATH = "routed"
PROFILE = os.path.join(ROOT, "profiles", "moe_layer_qwen3_30b_a3b_T64.md")
FFN_SOURCE = os.path.join(ROOT, "paper_2607_00466_amd", "csrc", "expert_ffn.hip")


def measured_traffic() -> int | None:
    """HBM bytes per FFN-up launch from the committed rocprofv3 counter profile
    (FETCH_SIZE + WRITE_SIZE, calibrated against a 1 GiB copy), or None when the
    kernel source has changed since the counters were taken."""
    import hashlib

    try:
        text = open(PROFILE).read()
    except OSError:
        return None
    fields = dict(l.split(": ", 1) for l in text.splitlines() if ": " in l and not l.startswith(("|", "#", "`")))
    src = hashlib.sha256(open(FFN_SOURCE, "rb").read()).hexdigest()[:16]
    if fields.get("expert_ffn_source_sha256_16", "").strip() != src:
        return None
    try:
        return int(float(fields["traffic_bytes_per_launch (ffn up, read + write)"]))
    except (KeyError, ValueError):
        return None


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def layer_bytes(shape: synth.LayerShape, T: int, U: int, gate: bool) -> int:
    """Algorithmic HBM bytes of one layer step: the union's expert weights,
    the gate (if routed by it), x in, out, and the routing ids and weights."""
    b = U * shape.expert_bytes + 4 * T * shape.H * 2 + 8 * T * shape.K
    if gate:
        b += 4 * shape.H * shape.E
    return b


def up_bytes(shape: synth.LayerShape, T: int, U: int) -> int:
    """Algorithmic bytes of one routed up launch: W1 and W3 of the union, x and the routing ids."""
    return U * 2 * shape.H * shape.I * 2 + 4 * T * shape.H + 4 * T * shape.K


def mx_matrix_bytes(shape: synth.LayerShape) -> int:
    """MXFP4 bytes of one H x I expert matrix: half a byte a value, one scale byte per 32."""
    return shape.H * shape.I // 2 + shape.H * shape.I // 32


def mx_layer_bytes(shape: synth.LayerShape, T: int, U: int, gate: bool) -> int:
    """layer_bytes with MXFP4 experts (codes and scales of W1, W3, W2)."""
    return layer_bytes(shape, T, U, gate) - U * shape.expert_bytes + U * 3 * mx_matrix_bytes(shape)


def mx_up_bytes(shape: synth.LayerShape, T: int, U: int) -> int:
    """Algorithmic bytes of one MXFP4 up launch: W1 and W3 codes and scales of the union, and x."""
    return U * 2 * mx_matrix_bytes(shape) + 4 * T * shape.H


class Bench:
    def __init__(self, shape: synth.LayerShape, T: int, seed: int = 0, share: "Bench | None" = None):
        """One layer at batch T.  With ``share``, the packed expert weights (and
        their rotation copies) of another bench of the same shape are reused."""
        self.shape = shape
        self.T = T
        self.d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
        self.x_np = synth.hidden_states(T, shape.H, seed)
        self.wg_np = synth.gate_weights(shape, seed)
        self.x = torch.from_numpy(self.x_np).cuda()
        self.wg = torch.from_numpy(self.wg_np).cuda()
        if share is not None:
            self.raw_weights = share.raw_weights
            self.weights = share.weights  # the same list: copies made by either are shared
        else:
            raw = synth.expert_weights(shape, seed, device="cuda")
            self.raw_weights = raw  # row-major, for the CPU baseline
            self.weights = [B.pack_expert_weights(*raw)]  # packed once, before any timing
        self.buf = B.LayerBuffers.allocate(self.d)
        self.stream = torch.cuda.current_stream()

    def rotate(self, union_bytes: int) -> None:
        R = max(2, math.ceil(ROTATE_BYTES / max(1, union_bytes)))
        R = min(R, 16)
        while len(self.weights) < R:
            self.weights.append(tuple(w.clone() for w in self.weights[0]))

    def step(self, i: int, routing=None, ev=None) -> None:
        w13, w2 = self.weights[i % len(self.weights)]
        d, b = self.d, self.buf
        # gate-bypassed routing is read in place by the bucket and the combine
        ids, w = (b.topk_ids, b.topk_w) if routing is None else routing
        if routing is None:
            B.moe_gate_topk(self.x, self.wg, d, b.logits, b.topk_ids, b.topk_w)
        if ev is not None:
            ev[0].record(self.stream)
        if FFN_PATH == "fused":
            # buckets, up and down projections (one launch up to 64 tokens)
            B.moe_expert_ffn_routed(self.x, w13, w2, ids, d, b.counts, b.offsets, b.perm_token,
                                    b.pair_pos, b.union_ids, b.union_size, b.y_perm, b.ws, b.sync)
            if ev is not None:
                ev[1].record(self.stream)
        else:
            if FFN_PATH == "routed":
                # buckets and the up projection (one launch up to 64 tokens, else two)
                B.moe_expert_ffn_up_routed(self.x, w13, ids, d, b.counts, b.offsets, b.perm_token,
                                           b.pair_pos, b.union_ids, b.union_size, b.ws)
            else:
                B.moe_bucket(ids, d, b.counts, b.offsets, b.perm_token, b.pair_pos, b.union_ids,
                             b.union_size)
                B.moe_expert_ffn_up(self.x, w13, b.offsets, b.perm_token, b.union_ids,
                                    b.union_size, d, b.ws)
            if ev is not None:
                ev[1].record(self.stream)
            B.moe_expert_ffn_down(b.ws, w2, b.offsets, b.perm_token, b.union_ids, b.union_size, d,
                                  b.y_perm)
        if ev is not None:
            ev[2].record(self.stream)
        B.moe_combine(b.y_perm, b.pair_pos, w, d, b.out)

    def union(self) -> int:
        torch.cuda.synchronize()
        return int(self.buf.union_size.item())

    def capture(self, steps: int, routing=None) -> "torch.cuda.CUDAGraph":
        """One HIP graph holding `steps` layer steps; step j uses weight copy j mod R."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for j in range(min(steps, len(self.weights))):
                self.step(j, routing)
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for j in range(steps):
                self.step(j, routing)
        torch.cuda.synchronize()
        return g

    def run_steps(self, n: int, full, per: int, tails: dict, routing=None) -> None:
        """Replay exactly n layer steps: n // per replays of the per-step graph, then one
        graph of the remaining n % per steps (captured on first use)."""
        for _ in range(n // per):
            full.replay()
        r = n % per
        if r:
            if r not in tails:
                tails[r] = self.capture(r, routing)
            tails[r].replay()

    def time(self, steps: int, warmup: int, routing=None) -> dict:
        # Whole layer: graph replays, so host launch cost stays out of the GPU
        # timeline.  A decode step runs its layers back to back inside one graph,
        # so a graph here holds several layer steps (a whole number of rotations
        # through the weight copies, at least LAYERS_PER_GRAPH): the per-replay
        # launch gap is paid once per graph, not once per layer.
        R = len(self.weights)
        per = R * max(1, math.ceil(LAYERS_PER_GRAPH / R))
        full = self.capture(per, routing)
        tails: dict = {}
        self.run_steps(warmup, full, per, tails, routing)
        if steps % per and steps % per not in tails:
            tails[steps % per] = self.capture(steps % per, routing)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(self.stream)
        self.run_steps(steps, full, per, tails, routing)
        t1.record(self.stream)
        torch.cuda.synchronize()
        layer_ms = t0.elapsed_time(t1) / steps
        # Spread: events between consecutive replays of the full graph (a
        # separate pass), each replay's time divided by its layer steps.
        n_rep = max(2, steps // per)
        rev = [torch.cuda.Event(enable_timing=True) for _ in range(n_rep + 1)]
        rev[0].record(self.stream)
        for i in range(n_rep):
            full.replay()
            rev[i + 1].record(self.stream)
        torch.cuda.synchronize()
        per_layer = np.array([rev[i].elapsed_time(rev[i + 1]) for i in range(n_rep)]) / per
        del full, tails
        # Per-kernel durations of the FFN halves, with events around each
        # launch on the stream it runs on (a separate eager pass, so the
        # events do not perturb the whole-layer timing above; the host runs
        # ahead of the GPU here, so the kernels still run back to back).
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        for i in range(steps):
            self.step(i, routing, evs[i])
        torch.cuda.synchronize()
        up = np.array([e[0].elapsed_time(e[1]) for e in evs])
        down = np.array([e[1].elapsed_time(e[2]) for e in evs])
        return {"layer_ms": layer_ms, "up_ms": float(up.mean()), "down_ms": float(down.mean()),
                "up_ms_median": float(np.median(up)), "down_ms_median": float(np.median(down)),
                "layer_ms_p10_p50_p90": [float(np.percentile(per_layer, q)) for q in (10, 50, 90)]}


class MxBench(Bench):
    """Bench with MXFP4 experts (packed by moe_pack_mxfp4_up / _down)."""

    def __init__(self, shape: synth.LayerShape, T: int, seed: int = 0):
        self.shape = shape
        self.T = T
        self.d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
        self.x = torch.from_numpy(synth.hidden_states(T, shape.H, seed)).cuda()
        self.wg = torch.from_numpy(synth.gate_weights(shape, seed)).cuda()
        q = synth.mxfp4_expert_weights(shape, seed, device="cuda")
        self.weights = [B.pack_mxfp4_expert_weights(q["w1"], q["w3"], q["w2"])]
        del q
        self.buf = B.LayerBuffers.allocate(self.d)
        self.stream = torch.cuda.current_stream()

    def rotate(self, union_bytes: int) -> None:
        R = min(16, max(2, math.ceil(ROTATE_BYTES / max(1, union_bytes))))
        while len(self.weights) < R:
            self.weights.append(tuple((c.clone(), s.clone()) for c, s in self.weights[0]))

    def step(self, i: int, routing=None, ev=None) -> None:
        up, down = self.weights[i % len(self.weights)]
        d, b = self.d, self.buf
        # gate-bypassed routing is read in place by the bucket and the combine
        ids, w = (b.topk_ids, b.topk_w) if routing is None else routing
        if routing is None:
            B.moe_gate_topk(self.x, self.wg, d, b.logits, b.topk_ids, b.topk_w)
        if ev is not None:
            ev[0].record(self.stream)
        if FFN_PATH == "fused":
            B.moe_expert_ffn_mxfp4_routed(self.x, up, down, ids, d, b.counts, b.offsets,
                                          b.perm_token, b.pair_pos, b.union_ids, b.union_size,
                                          b.y_perm, b.ws, b.sync)
            if ev is not None:
                ev[1].record(self.stream)
        else:
            if FFN_PATH == "routed":
                B.moe_expert_ffn_mxfp4_up_routed(self.x, up, ids, d, b.counts, b.offsets,
                                                 b.perm_token, b.pair_pos, b.union_ids,
                                                 b.union_size, b.ws)
            else:
                B.moe_bucket(ids, d, b.counts, b.offsets, b.perm_token, b.pair_pos, b.union_ids,
                             b.union_size)
                B.moe_expert_ffn_mxfp4_up(self.x, up, b.offsets, b.perm_token, b.union_ids,
                                          b.union_size, d, b.ws)
            if ev is not None:
                ev[1].record(self.stream)
            B.moe_expert_ffn_mxfp4_down(b.ws, down, b.offsets, b.perm_token, b.union_ids,
                                        b.union_size, d, b.y_perm)
        if ev is not None:
            ev[2].record(self.stream)
        B.moe_combine(b.y_perm, b.pair_pos, w, d, b.out)


def mxfp4_point(steps: int, warmup: int) -> dict:
    """The gpt-oss-120b-shaped layer (E=128, top-4, H=I=2880) at T=256 with
    MXFP4 experts, gate-routed: the MXFP4 widening's figures for the bench
    line (layer and up-kernel time, GB/s and fraction of HBM peak)."""
    shape = synth.SHAPES["gpt_oss_120b"]
    T = 256
    log("gpt-oss MXFP4 layer for the bench line: building (synthetic weights, quantized to MXFP4)")
    bench = MxBench(shape, T)
    bench.step(0)
    U = bench.union()
    bench.rotate(U * 3 * mx_matrix_bytes(shape))
    r = bench.time(steps, warmup)
    lb = mx_layer_bytes(shape, T, U, True)
    ub = mx_up_bytes(shape, T, U)
    rec = {"workload": "gpt_oss_120b moe layer, T=256, gate-routed, MXFP4 experts", "U": U,
           "layer_us": round(r["layer_ms"] * 1e3, 2), "ffn_up_us": round(r["up_ms"] * 1e3, 2),
           "ffn_down_us": round(r["down_ms"] * 1e3, 2),
           "layer_GBps": round(lb / r["layer_ms"] / 1e6, 1),
           "layer_frac_of_hbm_peak": round(lb / r["layer_ms"] / 1e6 / HBM_PEAK_GBS, 4),
           "ffn_up_GBps": round(ub / r["up_ms"] / 1e6, 1),
           "ffn_up_frac_of_hbm_peak": round(ub / r["up_ms"] / 1e6 / HBM_PEAK_GBS, 4),
           "weight_copies": len(bench.weights)}
    log(f"gpt-oss MXFP4 gate-routed: U={U} layer {rec['layer_us']:.1f} us, up {rec['ffn_up_us']:.1f} us "
        f"({rec['ffn_up_GBps']:.0f} GB/s)")
    del bench
    torch.cuda.empty_cache()
    return rec


def mxfp4_workload(path: str, steps: int, warmup: int, layers: int = 36,
                   cases=(None, 32, 128), formats=("mxfp4", "bf16")) -> None:
    """One gpt-oss-120b-shaped layer (E=128, top-4, H=I=2880), T=256, with MXFP4
    experts beside the same layer with bf16 experts: gate-routed and controlled
    unions 32 and 128.  Then a decode step of ``layers`` distinct MXFP4 layers,
    all resident (1.7 GB each), gate-routed."""
    shape = synth.SHAPES["gpt_oss_120b"]
    T = 256
    res = {}
    with open(path, "a") as f:
        for fmt, cls in (("mxfp4", MxBench), ("bf16", Bench)):
            if fmt not in formats:
                continue
            log(f"gpt-oss {fmt}: building the layer (synthetic weights"
                f"{', quantized to MXFP4' if fmt == 'mxfp4' else ''})")
            bench = cls(shape, T)
            for U in cases:
                log(f"gpt-oss {fmt}: timing {'gate-routed' if U is None else f'controlled U={U}'}")
                routing = None
                if U is not None:
                    ids, w, _ = synth.controlled_routing(T, shape.E, shape.K, U, seed=0)
                    routing = (torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda())
                bench.step(0, routing)
                Ur = bench.union()
                ebytes = 3 * mx_matrix_bytes(shape) if fmt == "mxfp4" else shape.expert_bytes
                bench.rotate(Ur * ebytes)
                r = bench.time(steps, warmup, routing)
                lb = (mx_layer_bytes if fmt == "mxfp4" else layer_bytes)(shape, T, Ur, U is None)
                ub = (mx_up_bytes if fmt == "mxfp4" else up_bytes)(shape, T, Ur)
                rec = {"workload": "gpt_oss_120b moe layer, T=256", "experts": fmt,
                       "routing": "gate" if U is None else f"controlled U={U}", "U": Ur,
                       "layer_us": r["layer_ms"] * 1e3, "up_us": r["up_ms"] * 1e3,
                       "down_us": r["down_ms"] * 1e3, "layer_bytes": lb,
                       "layer_GBps": lb / r["layer_ms"] / 1e6,
                       "up_GBps": ub / r["up_ms"] / 1e6,
                       "weight_copies": len(bench.weights)}
                rec["layer_frac_of_hbm_peak"] = rec["layer_GBps"] / HBM_PEAK_GBS
                rec["up_frac_of_hbm_peak"] = rec["up_GBps"] / HBM_PEAK_GBS
                res[(fmt, U)] = rec
                f.write(json.dumps(rec) + "\n")
                f.flush()
                log(f"gpt-oss {fmt} {rec['routing']}: U={Ur} layer {rec['layer_us']:.1f} us "
                    f"({rec['layer_GBps']:.0f} GB/s), up {rec['up_us']:.1f} us ({rec['up_GBps']:.0f} GB/s), "
                    f"down {rec['down_us']:.1f} us")
            del bench
            torch.cuda.empty_cache()
        for U in cases if len(formats) == 2 else ():
            a, b = res[("mxfp4", U)], res[("bf16", U)]
            f.write(json.dumps({"workload": "gpt_oss_120b moe layer, T=256", "summary": True,
                                "routing": a["routing"], "U": a["U"],
                                "mxfp4_speedup_over_bf16": b["layer_us"] / a["layer_us"],
                                "byte_ratio": b["layer_bytes"] / a["layer_bytes"]}) + "\n")
        if layers <= 0:
            return
        # a whole decode step of distinct MXFP4 layers, every layer resident
        d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
        lay = []
        for l in range(layers):
            q = synth.mxfp4_expert_weights(shape, 0, l, device="cuda")
            packed = B.pack_mxfp4_expert_weights(q["w1"], q["w3"], q["w2"])
            del q
            x = torch.from_numpy(synth.hidden_states(T, shape.H, 0, l)).cuda()
            wg = torch.from_numpy(synth.gate_weights(shape, 0, l)).cuda()
            lay.append((x, wg, packed, B.LayerBuffers.allocate(d)))
        torch.cuda.synchronize()
        log(f"gpt-oss mxfp4: {layers} layers resident")

        def run_step():
            for x, wg, (up, down), buf in lay:
                B.moe_layer_mxfp4(x, wg, up, down, d, buf, path=FFN_PATH)

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            run_step()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run_step()
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        unions = [int(buf.union_size.item()) for *_, buf in lay]
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(5):
            g.replay()
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / 5
        step_bytes = sum(mx_layer_bytes(shape, T, u, True) for u in unions)
        rec = {"workload": f"gpt_oss_120b x{layers} layers (all resident), T=256, MXFP4 experts",
               "routing": "gate", "step_ms": ms, "mean_union": float(np.mean(unions)),
               "step_GBps": step_bytes / ms / 1e6}
        f.write(json.dumps(rec) + "\n")
        log(f"gpt-oss mxfp4 x{layers}: {ms:.3f} ms/step, mean union {rec['mean_union']:.1f}, "
            f"{rec['step_GBps']:.0f} GB/s")
        del g, lay
        torch.cuda.empty_cache()


def calibration(reps: int = 10) -> dict:
    """What plain streaming achieves on this GPU, for context beside the 8 TB/s peak:
    the library's streaming-read probe over 2 GiB (reads only) and a 2 GiB
    device-to-device copy (reads + writes), best of `reps`, HIP events on the
    current stream."""
    n = (2 << 30) // 4
    a = torch.ones(n, device="cuda")
    b = torch.empty_like(a)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")

    def best(fn) -> float:
        fn()
        torch.cuda.synchronize()
        t = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1))
        return min(t)

    read_ms = best(lambda: B.moe_stream_read_probe(a, sink))
    copy_ms = best(lambda: b.copy_(a))
    del a, b
    torch.cuda.empty_cache()
    return {"stream_read_GBps": round(4 * n / read_ms / 1e6, 1),
            "copy_GBps_read_plus_write": round(8 * n / copy_ms / 1e6, 1),
            "how": "best of 10: moe_stream_read_probe (non-temporal loads) over 2 GiB; a 2 GiB device copy"}


def cpu_baseline(bench: Bench, U: int, budget_s: float, threads: int = 1) -> dict:
    """The float64 oracle on the host, `threads` BLAS threads, on the same layer."""
    from threadpoolctl import threadpool_limits

    from oracle import moe_oracle

    w1, w3, w2 = (synth.bf16_bits(w) for w in bench.raw_weights)
    runs, t_total = 0, 0.0
    with threadpool_limits(limits=threads):
        while t_total < budget_s and runs < 50:
            t = time.perf_counter()
            moe_oracle.moe_layer(bench.x_np, bench.wg_np, w1, w3, w2, bench.shape.K)
            t_total += time.perf_counter() - t
            runs += 1
    per_layer = t_total / runs
    return {
        "value": layer_bytes(bench.shape, bench.T, U, True) / per_layer / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{runs} runs of the whole gate-routed layer (same inputs), float64 NumPy, "
                  f"{per_layer * 1e3:.0f} ms per layer, {os.cpu_count()} host cores visible",
    }


def host_threads() -> int:
    """Threads the host lets this process use (its affinity), at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


UNION_SWEEP = (16, 32, 64, 96, 128)       # controlled unions at T = 64
BATCH_SWEEP = (8, 16, 32, 64, 128, 256)   # decode batches at U = 32


def controlled_point(bench: "Bench", U: int, steps: int, warmup: int) -> dict:
    """Time the layer at batch bench.T with a controlled union of U experts
    (gate bypassed); bytes and rates count the realised union."""
    shape, T = bench.shape, bench.T
    ids, w, _ = synth.controlled_routing(T, shape.E, shape.K, U, seed=0)
    routing = (torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda())
    bench.step(0, routing)
    Ur = bench.union()
    bench.rotate(Ur * shape.expert_bytes)
    r = bench.time(steps, warmup, routing)
    lb = layer_bytes(shape, T, Ur, False)
    rec = {"T": T, "U_nominal": U, "U": Ur, "layer_us": round(r["layer_ms"] * 1e3, 2),
           "layer_GBps": round(lb / r["layer_ms"] / 1e6, 1),
           "frac_of_peak": round(lb / r["layer_ms"] / 1e6 / HBM_PEAK_GBS, 4),
           "up_us": round(r["up_ms"] * 1e3, 2), "down_us": round(r["down_ms"] * 1e3, 2),
           "up_frac_of_peak": round(up_bytes(shape, T, Ur) / r["up_ms"] / 1e6 / HBM_PEAK_GBS, 4)}
    log(f"T={T} U={Ur}: layer {rec['layer_us']:.1f} us ({rec['layer_GBps']:.0f} GB/s, "
        f"{100 * rec['frac_of_peak']:.1f}% of peak), up {rec['up_us']:.1f} us, down {rec['down_us']:.1f} us")
    return rec


def sweep(steps: int, warmup: int, path: str = "") -> dict:
    """The paper's motivating measurement on this layer (Motivation, "Active
    Expert Count Drives MoE Decode Latency"): latency against the union at a
    fixed batch (T = 64, U = 16 .. 128), and against the batch at a fixed union
    (U = 32, T = 8 .. 256), with a least-squares fit t = a + b U over the first.
    All points share one weight set (and its rotation copies)."""
    shape = synth.SHAPES["qwen3_30b_a3b"]
    base = Bench(shape, 64)
    union_pts = [controlled_point(base, U, steps, warmup) for U in UNION_SWEEP]
    batch_pts = []
    for T in BATCH_SWEEP:
        if T == 64:  # the union sweep's U = 32 point is this batch point
            batch_pts.append(next(r for r in union_pts if r["U_nominal"] == 32))
            continue
        bench = Bench(shape, T, share=base)
        batch_pts.append(controlled_point(bench, 32, steps, warmup))
        del bench
    del base
    torch.cuda.empty_cache()
    Us = np.array([r["U"] for r in union_pts], float)
    ts = np.array([r["layer_us"] for r in union_pts], float)
    b, a = np.polyfit(Us, ts, 1)
    r2 = 1 - ((ts - (a + b * Us)) ** 2).sum() / ((ts - ts.mean()) ** 2).sum()
    t64 = next(r["layer_us"] for r in batch_pts if r["T"] == 64)
    out = {"union_sweep_T64": union_pts, "batch_sweep_U32": batch_pts,
           "fit": {"model": "layer_us = a + b * U (union sweep)", "a_us": round(a, 2),
                   "b_us_per_expert": round(b, 4), "r2": round(r2, 5),
                   "per_expert_GBps": round(shape.expert_bytes / b / 1e3, 1),
                   "intercept_in_experts": round(a / b, 1)},
           # the paper's motivating figure, context only: on one MI300X with
           # vLLM's MoE kernels the layer's latency rises 4.7x as the active
           # experts go from 16 to 128 at decode batch 64
           "latency_ratio_largest_union_over_U16": round(ts[-1] / ts[0], 3),
           "paper_ratio_16_to_128": 4.7,
           "batch_flatness_T256_over_T64": round(
               next(r["layer_us"] for r in batch_pts if r["T"] == 256) / t64, 3)}
    log(f"fit: t = {a:.2f} + {b:.3f} U us (R^2 {r2:.4f}); ratio U={int(Us[-1])}/U=16 "
        f"{out['latency_ratio_largest_union_over_U16']:.2f} (paper, MI300X: 4.7)")
    if path:
        with open(path, "w") as f:
            for rec in union_pts + batch_pts:
                f.write(json.dumps(rec) + "\n")
            f.write(json.dumps({k: v for k, v in out.items() if not k.endswith(("T64", "U32"))}) + "\n")
    return out


class MultiLayer:
    """A decode step over many distinct MoE layers (packed weights resident in HBM).

    ``n_resident`` distinct layers are allocated; a step of ``n_layers`` layers
    cycles through them (each layer's weights far exceed the Infinity Cache,
    so a cycled layer is still read from HBM).
    """

    def __init__(self, shape: synth.LayerShape, T: int, n_layers: int, n_resident: int, seed: int = 0):
        self.shape, self.T, self.n_layers = shape, T, n_layers
        self.d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
        self.layers = []
        for layer in range(n_resident):
            raw = synth.expert_weights(shape, seed, layer, device="cuda")
            packed = B.pack_expert_weights(*raw)
            del raw
            x = torch.from_numpy(synth.hidden_states(T, shape.H, seed, layer)).cuda()
            wg = torch.from_numpy(synth.gate_weights(shape, seed, layer)).cuda()
            self.layers.append((x, wg, packed))
        torch.cuda.synchronize()
        self.bufs = [B.LayerBuffers.allocate(self.d) for _ in range(n_layers)]

    def step(self, routing=None) -> None:
        """One decode step; routing[l] = (ids, w) device tensors, or None for the gate."""
        for l in range(self.n_layers):
            x, wg, (w13, w2) = self.layers[l % len(self.layers)]
            r = None if routing is None else routing[l]
            B.moe_layer(x, wg, w13, w2, self.d, self.bufs[l], routing=r, path=FFN_PATH)

    def unions(self) -> list[int]:
        torch.cuda.synchronize()
        return [int(b.union_size.item()) for b in self.bufs]

    def time(self, steps: int, warmup: int, routing=None) -> float:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.step(routing)
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step(routing)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(steps):
            g.replay()
        t1.record()
        torch.cuda.synchronize()
        del g
        return t0.elapsed_time(t1) / steps


def domain_workload(path: str, steps: int, warmup: int) -> None:
    """48 Qwen3-30B-A3B-shaped layers per step, T=128, domain-clustered routing:
    a same-domain batch per domain vs a batch mixed evenly over the 8 domains."""
    shape = synth.SHAPES["qwen3_30b_a3b"]
    model = synth.DomainModel()
    L, T = 48, 128
    ml = MultiLayer(shape, T, L, L)
    subsets = synth.domain_subsets(model, L, seed=0)
    batches = synth.domain_batches(model, T)
    results = {}
    with open(path, "a") as f:
        for name, doms in batches.items():
            routing = []
            for l in range(L):
                ids, w = synth.domain_routing(model, subsets, doms, l, seed=0)
                routing.append((torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda()))
            ml.step(routing)
            us = ml.unions()
            ms = ml.time(steps, warmup, routing)
            step_bytes = sum(layer_bytes(shape, T, u, False) for u in us)
            rec = {"workload": "qwen3_30b_a3b x48 layers, T=128, domain-clustered", "batch": name,
                   "step_ms": ms, "mean_union": float(np.mean(us)), "unions": us,
                   "step_GBps": step_bytes / ms / 1e6}
            results[name] = rec
            f.write(json.dumps(rec) + "\n")
            f.flush()
            log(f"domains {name}: {ms:.3f} ms/step, mean union {np.mean(us):.1f}, {rec['step_GBps']:.0f} GB/s")
        same = [results[k] for k in results if k.startswith("same_")]
        summary = {"workload": "qwen3_30b_a3b x48 layers, T=128, domain-clustered", "summary": True,
                   "same_domain_mean_step_ms": float(np.mean([r["step_ms"] for r in same])),
                   "same_domain_mean_union": float(np.mean([r["mean_union"] for r in same])),
                   "mixed_step_ms": results["mixed"]["step_ms"],
                   "mixed_mean_union": results["mixed"]["mean_union"]}
        summary["union_reduction"] = 1 - summary["same_domain_mean_union"] / summary["mixed_mean_union"]
        summary["step_time_reduction"] = 1 - summary["same_domain_mean_step_ms"] / summary["mixed_step_ms"]
        f.write(json.dumps(summary) + "\n")
        log(f"domains: same-domain batches use {100 * summary['union_reduction']:.1f}% fewer experts per layer "
            f"and {100 * summary['step_time_reduction']:.1f}% less step time than the mixed batch")
    del ml
    torch.cuda.empty_cache()


def gpt_oss_workload(path: str, steps: int, warmup: int, resident: int = 20) -> None:
    """36 gpt-oss-120b-shaped layers per step (bf16), T=256, gate-routed and
    controlled unions 32 and 128.  ``resident`` distinct layers are allocated
    (6.37 GB each) and cycled."""
    shape = synth.SHAPES["gpt_oss_120b"]
    L, T = 36, 256
    ml = MultiLayer(shape, T, L, resident)
    with open(path, "a") as f:
        for U in (None, 32, 128):
            routing = None
            if U is not None:
                routing = []
                for l in range(L):
                    ids, w, _ = synth.controlled_routing(T, shape.E, shape.K, U, seed=0, layer=l)
                    routing.append((torch.from_numpy(ids).cuda(), torch.from_numpy(w).cuda()))
            ml.step(routing)
            us = ml.unions()
            ms = ml.time(steps, warmup, routing)
            step_bytes = sum(layer_bytes(shape, T, u, routing is None) for u in us)
            rec = {"workload": f"gpt_oss_120b x{L} layers ({resident} resident, cycled), T=256",
                   "routing": "gate" if U is None else f"controlled U={U}", "step_ms": ms,
                   "mean_union": float(np.mean(us)), "step_GBps": step_bytes / ms / 1e6}
            f.write(json.dumps(rec) + "\n")
            f.flush()
            log(f"gpt-oss {rec['routing']}: {ms:.3f} ms/step, mean union {rec['mean_union']:.1f}, "
                f"{rec['step_GBps']:.0f} GB/s")
    del ml
    torch.cuda.empty_cache()


def signature_workload(path: str, reps: int = 20) -> None:
    """The expert-signature cache at the paper's largest shape (48 MoE layers,
    E=128, top-8): capture of one 2048-token prefill forward into 16-token
    blocks of a 4096-block cache, and the per-request sums of 64 requests of
    64 blocks.  GPU times are graph replays; the oracle runs the same capture
    and sums on one host thread."""
    from oracle import signature as SO

    L, E, K, T, BS, NB, R = 48, 128, 8, 2048, 16, 4096, 64
    rng = np.random.default_rng(0)
    ids_np = synth.prefill_picks(L, T, E, K, seed=0, skew=1.1)
    table_np = rng.permutation(NB)[:T // BS].astype(np.int32)
    tb_np = table_np[np.arange(T) // BS]
    ids = torch.from_numpy(ids_np).cuda()
    tb = torch.from_numpy(tb_np).cuda()
    blocks = torch.from_numpy(table_np).cuda()
    sig = torch.zeros((NB, L, E), dtype=torch.int8, device="cuda")
    req_table = torch.from_numpy(rng.integers(0, NB, (R, 64)).astype(np.int32)).cuda()
    req_n = torch.full((R,), 64, dtype=torch.int32, device="cuda")
    out = torch.empty((R, L, E), dtype=torch.int32, device="cuda")

    def timed(fn) -> float:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(10):
                fn()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / (10 * reps) * 1e3  # us per call

    reset_us = timed(lambda: B.moe_sig_reset(blocks, sig))
    pair_us = timed(lambda: (B.moe_sig_reset(blocks, sig), B.moe_sig_capture(ids, tb, 0, L, E, sig)))
    capture_us = pair_us - reset_us
    counts_us = timed(lambda: B.moe_sig_request_counts(sig, req_table, req_n, out))
    picks = L * T * K
    t0 = time.perf_counter()
    ref, _ = SO.capture(SO.new_cache(NB, L, E), ids_np, tb_np)
    cpu_capture_s = time.perf_counter() - t0
    t0 = time.perf_counter()
    tabs = req_table.cpu().numpy()
    for r in range(R):
        SO.request_counts(ref, tabs[r])
    cpu_counts_s = time.perf_counter() - t0
    # correctness of what was timed
    B.moe_sig_reset(blocks, sig)
    B.moe_sig_capture(ids, tb, 0, L, E, sig)
    torch.cuda.synchronize()
    ok = bool(np.array_equal(sig.cpu().numpy().astype(np.int64), ref))
    counts_bytes = R * 64 * L * E + 4 * R * L * E
    recs = [
        {"workload": "signature capture: 48 layers, E=128, top-8, one 2048-token prefill, 16-token blocks",
         "call": "moe_sig_capture", "us": round(capture_us, 2), "picks": picks,
         "Gpicks_per_s": round(picks / capture_us / 1e3, 2),
         "cpu_oracle": {"us": round(cpu_capture_s * 1e6), "cores": 1}, "matches_oracle": ok},
        {"workload": "signature sums: 64 requests x 64 blocks, 48 layers, E=128",
         "call": "moe_sig_request_counts", "us": round(counts_us, 2),
         "GBps": round(counts_bytes / counts_us / 1e3, 1),
         "roofline": {"bound": "hbm", "achieved": round(counts_bytes / counts_us / 1e3, 1),
                      "peak": HBM_PEAK_GBS, "unit": "GB/s",
                      "frac": round(counts_bytes / counts_us / 1e3 / HBM_PEAK_GBS, 4)},
         "cpu_oracle": {"us": round(cpu_counts_s * 1e6), "cores": 1}},
        {"workload": "signature reset: 128 blocks of 6 KiB", "call": "moe_sig_reset",
         "us": round(reset_us, 2)},
    ]
    with open(path, "a") as f:
        for rec in recs:
            f.write(json.dumps(rec) + "\n")
            log(f"signature {rec['call']}: {rec['us']} us")


def routing_workload(path: str, workers: int = 16, per_worker: int = 64, layers_timed: int = 8) -> None:
    """ELDR end to end on synthetic domain traffic (Design: Expert Signature,
    Offline clustering, Online routing), against round-robin.

    1024 calibration requests (8 domains, 48 MoE layers, E=128, top-8) give
    prefill counts and decode activation probabilities; the native library
    fits the IDF table, the greedy layer mask and a Hungarian-balanced
    K-means with one centroid per worker.  Then workers * per_worker new
    requests are routed by locality-band routing (tau = 0.1) and by
    round-robin; each worker's decode step (one token per request) is drawn
    from its requests' domains, and its union per layer is counted.  Finally
    each worker's step is run on the GPU for `layers_timed` layers through
    the MoE layer (Qwen3-30B-A3B-shaped weights, controlled routing = the
    drawn picks) and timed."""
    model = synth.DomainModel()
    L, E, K, N_cal, pre_tok, dec_tok = 48, model.E, model.K, 1024, 32, 16
    subsets = synth.domain_subsets(model, L, seed=0)

    def counts_of(ids):  # ids [L, R, T, K] -> counts [R, L, E]
        R = ids.shape[1]
        out = np.zeros((R, L, E), np.int32)
        for layer in range(L):
            for r in range(R):
                out[r, layer] = np.bincount(ids[layer, r].ravel(), minlength=E)
        return out

    rng = np.random.default_rng(7)
    cal_dom = rng.integers(0, model.n_domains, N_cal)
    cal_counts = counts_of(synth.domain_requests(model, subsets, cal_dom, pre_tok, seed=1, stream=0))
    P = counts_of(synth.domain_requests(model, subsets, cal_dom, dec_tok, seed=1, stream=1)).reshape(N_cal, -1)
    P = (P / np.linalg.norm(P, axis=1, keepdims=True)).astype(np.float32)
    pairs = rng.choice(N_cal, (4000, 2))
    pairs = pairs[pairs[:, 0] != pairs[:, 1]]
    t0 = time.perf_counter()
    idf = B.eldr_idf(cal_counts)
    order, curve, n_star = B.eldr_greedy_layers(cal_counts, idf, P, pairs)
    mask = order[:n_star].tolist()
    S_cal = np.stack([B.eldr_signature(c, idf, mask) for c in cal_counts])
    init = rng.choice(N_cal, workers, replace=False)
    C, _, iters = B.eldr_balanced_kmeans(S_cal, workers, init, max_iters=50)
    fit_s = time.perf_counter() - t0
    log(f"routing: offline fit {fit_s:.2f} s (N*={n_star} of {L} layers, rho {curve[n_star - 1]:.3f}, "
        f"k-means {iters} iterations)")

    R = workers * per_worker
    dom = rng.integers(0, model.n_domains, R)
    req_counts = counts_of(synth.domain_requests(model, subsets, dom, pre_tok, seed=2, stream=0))
    S = np.stack([B.eldr_signature(c, idf, mask) for c in req_counts])
    t0 = time.perf_counter()
    eldr_w, eldr_loads = B.eldr_route_batch(S, C, np.zeros(workers, np.int32), 0.1)
    route_us = (time.perf_counter() - t0) / R * 1e6
    rr_w = np.arange(R) % workers
    step = synth.domain_requests(model, subsets, dom, 1, seed=2, stream=2)[:, :, 0, :]  # [L, R, K]

    shape = synth.SHAPES["qwen3_30b_a3b"]
    raw = synth.expert_weights(shape, 0, 0, device="cuda")
    packed = [B.pack_expert_weights(*raw)]
    packed.append(tuple(w.clone() for w in packed[0]))
    del raw
    wg = torch.from_numpy(synth.gate_weights(shape, 0, 0)).cuda()
    def measure(assign):
        unions = np.zeros((workers, L))
        sizes = np.bincount(assign, minlength=workers)
        for w in range(workers):
            members = np.nonzero(assign == w)[0]
            for layer in range(L):
                unions[w, layer] = len(np.unique(step[layer, members]))
        # GPU: each worker's step over the first layers_timed layers
        worker_us = []
        for w in range(workers):
            members = np.nonzero(assign == w)[0]
            T = len(members)
            if T == 0:
                worker_us.append(0.0)
                continue
            d = B.dims(T, shape.H, shape.E, shape.K, shape.I)
            buf = B.LayerBuffers.allocate(d)
            x = torch.from_numpy(synth.hidden_states(T, shape.H, 0, w)).cuda()
            routes = []
            for layer in range(layers_timed):
                ids = torch.from_numpy(np.ascontiguousarray(step[layer, members])).cuda()
                wts = torch.from_numpy(synth.dirichlet_weights(T, K, np.random.default_rng(layer))).cuda()
                routes.append((ids, wts))

            def run():
                for layer in range(layers_timed):
                    w13, w2 = packed[layer % 2]
                    B.moe_layer(x, wg, w13, w2, d, buf, routing=routes[layer], path=FFN_PATH)

            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                run()
            torch.cuda.current_stream().wait_stream(side)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run()
            g.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(10):
                g.replay()
            e1.record()
            torch.cuda.synchronize()
            worker_us.append(e0.elapsed_time(e1) / 10 * 1e3)
            del g, buf
        return {"mean_union": float(unions.mean()), "max_batch": int(sizes.max()),
                "min_batch": int(sizes.min()),
                "mean_worker_step_us": float(np.mean(worker_us)),
                "max_worker_step_us": float(np.max(worker_us))}

    e, r = measure(eldr_w), measure(rr_w)
    rec = {"workload": f"ELDR vs round-robin: {workers} workers x {per_worker} requests, 8 synthetic domains, "
                       f"48 MoE layers (E=128, top-8); decode step timed on {layers_timed} Qwen3-30B-A3B-shaped layers",
           "fit_s": round(fit_s, 2), "n_star": n_star, "rho": round(float(curve[n_star - 1]), 4),
           "kmeans_iterations": iters, "route_us_per_request": round(route_us, 2),
           "eldr": e, "round_robin": r,
           "union_reduction": round(1 - e["mean_union"] / r["mean_union"], 4),
           "mean_step_reduction": round(1 - e["mean_worker_step_us"] / r["mean_worker_step_us"], 4),
           "max_step_reduction": round(1 - e["max_worker_step_us"] / r["max_worker_step_us"], 4)}
    with open(path, "a") as f:
        f.write(json.dumps(rec) + "\n")
    log(f"routing: union per worker-layer {e['mean_union']:.1f} (ELDR) vs {r['mean_union']:.1f} (RR): "
        f"{100 * rec['union_reduction']:.1f}% fewer; worker decode step {e['mean_worker_step_us']:.0f} vs "
        f"{r['mean_worker_step_us']:.0f} us ({100 * rec['mean_step_reduction']:.1f}% less); batch sizes "
        f"{e['min_batch']}-{e['max_batch']} (ELDR)")
    del packed
    torch.cuda.empty_cache()


def main() -> int:
    global FFN_PATH
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="host time budget of the CPU-oracle baseline (0 to skip)")
    ap.add_argument("--sweep", default="",
                    help="also write the union and batch sweeps (which the bench line carries) to this file")
    ap.add_argument("--no-sweep", action="store_true",
                    help="leave the union and batch sweeps out of the bench line")
    ap.add_argument("--no-mxfp4-line", action="store_true",
                    help="leave the gate-routed gpt-oss MXFP4 layer out of the bench line")
    ap.add_argument("--point", action="append", default=[],
                    help="T:U -- time only this controlled-union point (repeatable; no bench line)")
    ap.add_argument("--signature", default="",
                    help="also time the expert-signature cache calls, appending JSON lines to this file")
    ap.add_argument("--signature-only", action="store_true",
                    help="run only the --signature measurement (no layer bench line)")
    ap.add_argument("--routing", default="",
                    help="also run ELDR routing vs round-robin end to end (native fit + routing, GPU "
                         "decode steps), appending a JSON line to this file")
    ap.add_argument("--routing-only", action="store_true",
                    help="run only the --routing measurement (no layer bench line)")
    ap.add_argument("--multilayer", default="",
                    help="also run the 48-layer domain-clustered and 36-layer gpt-oss workloads, "
                         "appending JSON lines to this file")
    ap.add_argument("--multilayer-only", action="store_true",
                    help="run only the --multilayer measurement (no layer bench line)")
    ap.add_argument("--multilayer-parts", default="domain,gpt_oss",
                    help="which --multilayer workloads to run: domain and/or gpt_oss")
    ap.add_argument("--mxfp4", default="",
                    help="also run the gpt-oss-shaped layer with MXFP4 experts beside bf16 experts "
                         "and a 36-layer MXFP4 step, appending JSON lines to this file")
    ap.add_argument("--mxfp4-only", action="store_true",
                    help="run only the --mxfp4 measurement (no layer bench line)")
    ap.add_argument("--mxfp4-cases", default="gate,32,128",
                    help="routings of the --mxfp4 layer: 'gate' and/or controlled union sizes")
    ap.add_argument("--mxfp4-formats", default="mxfp4,bf16", help="expert formats of the --mxfp4 layer")
    ap.add_argument("--ffn-path", default=FFN_PATH, choices=B.FFN_PATHS,
                    help="how a layer step runs the expert FFN: one launch (fused), buckets + up "
                         "then down (routed), or bucket, up, down (split)")
    ap.add_argument("--mxfp4-layers", type=int, default=36,
                    help="layers of the --mxfp4 multi-layer step (0 to skip it)")
    args = ap.parse_args()
    FFN_PATH = args.ffn_path
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the layer runs on one GPU and has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        return 2
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    B.load()
    mx_args = dict(layers=args.mxfp4_layers, formats=tuple(args.mxfp4_formats.split(",")),
                   cases=tuple(None if c == "gate" else int(c) for c in args.mxfp4_cases.split(",")))
    if args.mxfp4_only:
        mxfp4_workload(args.mxfp4 or "mxfp4.jsonl", args.steps, args.warmup, **mx_args)
        return 0
    if args.point:
        shape = synth.SHAPES["qwen3_30b_a3b"]
        base = None
        for spec in args.point:
            T, U = (int(v) for v in spec.split(":"))
            bench = Bench(shape, T, share=base)
            base = base or bench
            print(json.dumps({"workload": "qwen3_30b_a3b moe layer, controlled union",
                              **controlled_point(bench, U, args.steps, args.warmup)}), flush=True)
        return 0
    if args.routing_only:
        routing_workload(args.routing or "routing.jsonl")
        return 0
    if args.signature_only:
        signature_workload(args.signature or "signature.jsonl")
        if args.routing:
            routing_workload(args.routing)
        return 0
    if args.multilayer_only:
        parts = args.multilayer_parts.split(",")
        if "domain" in parts:
            domain_workload(args.multilayer or "multilayer.jsonl", 10, 2)
        if "gpt_oss" in parts:
            gpt_oss_workload(args.multilayer or "multilayer.jsonl", 5, 1)
        return 0
    shape = synth.SHAPES["qwen3_30b_a3b"]
    T = 64
    bench = Bench(shape, T)
    bench.step(0)
    U = bench.union()
    bench.rotate(U * shape.expert_bytes)
    log(f"workload qwen3_30b_a3b T={T}: union {U}, {len(bench.weights)} weight copies")
    r = bench.time(args.steps, args.warmup)
    lb = layer_bytes(shape, T, U, True)
    value = lb / r["layer_ms"] / 1e6
    ub = up_bytes(shape, T, U)
    achieved = ub / r["up_ms"] / 1e6
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["layer_ms"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "qwen3_30b_a3b moe layer, decode batch 64, gate-routed",
                   "E": shape.E, "top_k": shape.K, "hidden": shape.H, "intermediate": shape.I,
                   "tokens": T, "union": U, "weight_copies": len(bench.weights)},
        "layer_us": round(r["layer_ms"] * 1e3, 2),
        "layer_us_p10_p50_p90": [round(v * 1e3, 2) for v in r["layer_ms_p10_p50_p90"]],
        "layer_frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "ffn_up_us": round(r["up_ms"] * 1e3, 2),
        "ffn_down_us": round(r["down_ms"] * 1e3, 2),
        "roofline": {"bound": "hbm", "kernel": "ffn_kernel<up, routed> (moe_expert_ffn_up_routed: buckets + up projection)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                     "bytes_per_launch": ub},
    }
    out["calibration"] = calibration()
    log(f"calibration: {out['calibration']}")
    if args.cpu_seconds > 0:
        log("timing the CPU oracle ...")
        out["cpu_baseline"] = cpu_baseline(bench, U, args.cpu_seconds)
        # secondary, for context: the same oracle with every host thread it may use
        n = host_threads()
        if n > 1:
            out["cpu_baseline_all_threads"] = cpu_baseline(bench, U, args.cpu_seconds / 2, threads=n)
    del bench
    torch.cuda.empty_cache()
    if not args.no_sweep:
        log("union and batch sweeps (controlled routing) ...")
        out["sweep"] = sweep(max(20, args.steps // 2), args.warmup, args.sweep)
    if not args.no_mxfp4_line:
        out["mxfp4_gpt_oss"] = mxfp4_point(max(20, args.steps // 4), args.warmup)
    if args.signature:
        signature_workload(args.signature)
    if args.routing:
        routing_workload(args.routing)
    if args.multilayer:
        parts = args.multilayer_parts.split(",")
        if "domain" in parts:
            domain_workload(args.multilayer, 10, 2)
        if "gpt_oss" in parts:
            gpt_oss_workload(args.multilayer, 5, 1)
    if args.mxfp4:
        mxfp4_workload(args.mxfp4, max(20, args.steps // 2), args.warmup, **mx_args)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
