#!/usr/bin/env python3
"""Benchmark of the FluxBin LUT-GEMV hot path on one MI355X.

Step = one pass of the hot path over one batch: the batch-1 LUT-GEMV of the 70B-shaped MLP layers up (28672x8192,
out x in) and down (8192x28672), 3 global bases + 1 salient base on 5% of the columns, mu = 8, one row scale per 128
columns, fp16 activations with 0.1% outlier channels. Synthetic seeded data (no weights are available); inputs are
packed and resident in HBM before timing. Several packed copies of each layer (> 2x the 256 MB Infinity Cache in
total) are rotated so that every launch streams its signs from HBM.

value = algorithmic bytes of the K steps / time of the K steps (GB/s). Algorithmic bytes per call:
  Kb*M*N/8 + Ks*M*S/8 (sign bits) + 2*Kb*M*ceil(N/g_r) + 2*Ks*M*ceil(S/g_s) (fp16 row scales)
  + 2*Kb*N + 2*Ks*S (fp16 column scales) + 2*S (16-bit salient indices) + 2*B*N (x) + 2*B*M (fp16 y).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time
from typing import Dict

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "achieved HBM GB/s (% of peak) + µs per LUT-GEMV, batch 1, 4096² and 8192×28672"
WORKLOAD = ("70B MLP up 28672x8192 + down 8192x28672 (out x in), Kb=3 + Ks=1 on 5% salient columns, mu=8, "
            "g_r=128, batch 1")


def algorithmic_bytes(spec, B: int = 1) -> int:
    M, N, Kb, Ks, S = spec.M, spec.N, spec.Kb, spec.Ks, spec.S
    sal = S if Ks > 0 else 0
    G_r = -(-N // spec.g_r)
    G_s = -(-S // spec.g_s) if sal else 0
    return (Kb * M * N // 8 + Ks * M * sal // 8 + 2 * Kb * M * G_r + 2 * Ks * M * G_s + 2 * Kb * N + 2 * Ks * sal
            + 2 * S + 2 * B * N + 2 * B * M)


def lookups(spec, B: int = 1) -> int:
    return B * spec.M * (spec.Kb * -(-spec.N // spec.mu) + spec.Ks * -(-spec.S // spec.mu))


# Every layer's launches rotate over distinct packed copies totalling at least this many bytes (over twice the 256 MB
# last-level cache), so that each launch reads its weights from HBM.
COPIES_BYTES_PER_LAYER = 600e6


class Bench:
    def __init__(self, layer_specs, B: int, copies_target_bytes: float, min_copies: int = 1, layers=None):
        import numpy as np
        import torch
        from paper_2608_15602_amd import fluxbin as fb
        from synth import make_activations, make_layer
        self.fb = fb
        self.specs = layer_specs
        self.B = B
        self.items = []
        for li, spec in enumerate(layer_specs):
            L = layers[li] if layers is not None else make_layer(spec)
            dev = {}
            for name in ("signs", "alpha_r", "alpha_c", "sal_idx", "sal_signs", "alpha_sr", "alpha_sc"):
                a = getattr(L, name)
                dt = {np.dtype(np.uint32): np.int32, np.dtype(np.uint16): np.int16, np.dtype(np.int32): np.int32}[
                    a.dtype]
                dev[name] = torch.from_numpy(np.ascontiguousarray(a).view(dt)).cuda()
            shape = fb.make_shape(spec.M, spec.N, spec.Kb, spec.Ks, spec.mu, spec.g_r, spec.S, spec.g_s)
            one = fb.fluxbin_pack_query(shape)
            n_copies = max(min_copies, math.ceil(copies_target_bytes / (one * len(layer_specs))))
            packs = [fb.fluxbin_pack(shape, dev) for _ in range(n_copies)]
            del dev
            x = torch.from_numpy(make_activations(L, B).view(np.float16)).cuda()
            y = torch.empty(B, spec.M, dtype=torch.float16, device="cuda")
            ws = fb.make_workspace(packs[0], B)
            self.items.append(dict(spec=spec, L=L, packs=packs, x=x, y=y, ws=ws,
                                   bytes=algorithmic_bytes(spec, B), lookups=lookups(spec, B)))
        torch.cuda.synchronize()

    def launch(self, it, step):
        p = it["packs"][step % len(it["packs"])]
        if self.B == 1:
            self.fb.fluxbin_lut_gemv(p, it["x"][0], y=it["y"][0], workspace=it["ws"])
        else:
            self.fb.fluxbin_lut_gemm_smallbatch(p, it["x"], y=it["y"], workspace=it["ws"])

    def graph(self, steps: int, start: int = 0, items=None):
        """Capture `steps` steps (every layer once per step, rotating packed copies) in one HIP graph."""
        import torch
        items = self.items if items is None else items
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                for s in range(steps):
                    for it in items:
                        self.launch(it, start + s)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        return g

    @staticmethod
    def time_graph(g, reps: int = 1):
        import torch
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    def run(self, steps: int, warmup: int, replays: int = 1):
        """Warmup steps, then a HIP graph of exactly `steps` steps, replayed `replays` times, each replay between two
        events on the replay stream (synchronized on both sides). Returns the milliseconds of every replay and the
        wall-clock seconds of all of them."""
        import torch
        for s in range(warmup):
            for it in self.items:
                self.launch(it, s)
        g = self.graph(steps, warmup)
        g.replay()          # first replay outside the timed region (graph upload)
        torch.cuda.synchronize()
        # the replays run back to back (an event between consecutive replays, no host synchronization until the
        # last one), so the device never idles inside the timed region; each replay is timed by its own event pair
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(replays + 1)]
        wall0 = time.perf_counter()
        ev[0].record()
        for r in range(replays):
            g.replay()
            ev[r + 1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        ms = [ev[r].elapsed_time(ev[r + 1]) for r in range(replays)]
        return ms, wall

    def per_launch_us(self, launches: int = 60, reps: int = 5):
        """Average duration of each layer's launch: a graph of `launches` launches of that layer alone (rotating
        copies), median of `reps` replays, divided by the launch count."""
        out = []
        for it in self.items:
            g = self.graph(launches, 0, [it])
            g.replay()
            ts = sorted(self.time_graph(g) * 1000.0 / launches for _ in range(reps))
            out.append(ts[len(ts) // 2])
        return out

    def stream_probe_us(self, launches: int = 60, reps: int = 5):
        """Average duration of the stream probe on each layer (the batch-1 kernel's weight requests, same launch plan,
        without the table work), timed like per_launch_us: the bandwidth this access pattern reaches on the device."""
        import torch
        sink = torch.zeros(256, dtype=torch.int32, device="cuda")
        out = []
        for it in self.items:
            g = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                with torch.cuda.graph(g, stream=side):
                    for s in range(launches):
                        self.fb.fluxbin_stream_probe(it["packs"][s % len(it["packs"])], sink)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            g.replay()
            ts = sorted(self.time_graph(g) * 1000.0 / launches for _ in range(reps))
            out.append(ts[len(ts) // 2])
        return out

    def set_batch(self, B: int):
        """Rebind activations, outputs and workspaces for batch B (the packed copies stay)."""
        import numpy as np
        import torch
        from synth import make_activations
        self.B = B
        for it in self.items:
            it["x"] = torch.from_numpy(make_activations(it["L"], B).view(np.float16)).cuda()
            it["y"] = torch.empty(B, it["spec"].M, dtype=torch.float16, device="cuda")
            it["ws"] = self.fb.make_workspace(it["packs"][0], B)
            it["bytes"] = algorithmic_bytes(it["spec"], B)
            it["lookups"] = lookups(it["spec"], B)
        torch.cuda.synchronize()

    def cold_launch_us(self, trials: int = 5):
        """Single eager launches, each event-timed on its own: the caches hold none of the packed copy it reads (the
        copies rotate and together exceed the 256 MB last-level cache), and the launch overhead is included. Median
        over `trials` per layer."""
        import torch
        out = []
        for it in self.items:
            ts = []
            for k in range(trials):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record()
                self.launch(it, 1 + k)
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1000.0)
            ts.sort()
            out.append(ts[len(ts) // 2])
        return out


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "k_gemv_b1_mlp70b_hbm_traffic.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_15602_amd", "csrc", f) for f in ("fluxbin_gemv.hip", "fluxbin_host.cpp", "fluxbin_device.h", "fluxbin_internal.h")]


def measured_traffic():
    """HBM bytes per launch of each layer from the committed counter summary (FETCH_SIZE and WRITE_SIZE passes scaled
    by a plain copy of known size), or None when the kernel or launch-plan sources changed since it was taken."""
    import hashlib
    try:
        text = open(TRAFFIC_PROFILE).read()
    except OSError:
        return None
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    sha = None
    per = {}
    for line in text.splitlines():
        if line.startswith("kernel_source_sha256:"):
            sha = line.split()[1]
        if line.startswith("traffic_bytes_per_launch:"):
            for kv in line.split(":", 1)[1].split():
                k, v = kv.split("=")
                per[k] = int(v)
    if sha != h.hexdigest() or not per:
        return None
    return per


def cpu_baseline(bench, budget_s: float):
    """The fp64 oracle (explicit reconstruction + matvec, untuned) on a bounded contiguous row sample of each layer;
    throughput scaled to the same algorithmic bytes per row as the GPU figure."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    done_bytes = 0.0
    t_total = 0.0
    parts = []
    for it in bench.items:
        spec = it["spec"]
        x = it["x"].cpu().numpy().view(np.uint16)
        # one 256-row probe to size the sample to the time budget
        t = time.perf_counter()
        oracle.gemv_dense(it["L"], x, row_range=(0, min(256, spec.M)))
        per_row = (time.perf_counter() - t) / min(256, spec.M)
        rows = int(min(spec.M, max(256, budget_s / len(bench.items) / per_row)))
        t = time.perf_counter()
        oracle.gemv_dense(it["L"], x, row_range=(0, rows))
        dt = time.perf_counter() - t
        t_total += dt
        done_bytes += it["bytes"] * rows / spec.M
        parts.append(f"{spec.name}: rows 0..{rows - 1} of {spec.M}")
    res = {"value": round(done_bytes / t_total / 1e9, 4), "unit": "GB/s", "cores": int(threads), "kind": "oracle",
           "sample": "; ".join(parts) + f" (fp64 reconstruct + matvec, {t_total:.1f} s)"}
    it = bench.items[0]
    spec = it["spec"]
    x = it["x"].cpu().numpy().view(np.uint16)
    # the same oracle on one core (BLAS limited to one thread), on a smaller sample of the first layer
    try:
        from threadpoolctl import threadpool_limits
        rows = 512
        with threadpool_limits(limits=1):
            t = time.perf_counter()
            oracle.gemv_dense(it["L"], x, row_range=(0, rows))
            dt = time.perf_counter() - t
        res["one_core"] = {"value": round(it["bytes"] * rows / spec.M / dt / 1e9, 4), "unit": "GB/s",
                           "sample": f"{spec.name}: rows 0..{rows - 1} ({dt:.1f} s)"}
    except Exception as e:   # threadpoolctl missing: report why
        res["one_core"] = {"value": None, "error": str(e)}
    # matvec only, on an already reconstructed fp64 block of W-hat (the reconstruction is not timed); 8192 rows of the
    # first layer are 0.5 GB, more than the host's last-level cache, so the matvecs stream it from memory
    rows = min(spec.M, 8192)
    W = oracle.reconstruct_rows(it["L"], 0, rows)
    xv = oracle.f16_to_f64(x)[0]
    reps = 0
    t = time.perf_counter()
    while time.perf_counter() - t < 2.0 or reps < 3:
        W @ xv
        reps += 1
    dt = (time.perf_counter() - t) / reps
    res["matvec_only"] = {"value": round(it["bytes"] * rows / spec.M / dt / 1e9, 4), "unit": "GB/s",
                          "sample": f"{spec.name}: fp64 rows 0..{rows - 1} reconstructed beforehand, {reps} matvecs",
                          "fp64_bytes_read_GBps": round(W.nbytes / dt / 1e9, 2)}
    del W
    try:
        with open("/proc/cpuinfo") as f:
            res["cpu_model"] = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
    except OSError:
        pass
    res["logical_cpus"] = os.cpu_count()
    return res


def small_batch_us(specs, batches, launches=40, rounds=3):
    """Per-call microseconds of the small-batch product on the same layers, graph-timed like the batch-1 figure, for
    the default kernel choice and, on the same packed copies, each kernel forced: the split-tile matrix-core kernel (the
    sign decode per bit is shared by all batch rows), the LUT batch kernel (batch-interleaved tables, each sign word
    read once for all batch rows) and, where a layer fits it, the row-complete matrix-core kernel. They are measured in
    turn, `rounds` times, and each figure is the median of its rounds (the first measurement of a process runs at lower
    clocks)."""
    import statistics
    import torch
    out = {}
    for B in batches:
        b = Bench(specs, B, COPIES_BYTES_PER_LAYER * len(specs))
        kernels = [("mfma", {"mfma": 1, "mfma_rows": 0}), ("lut", {"mfma": 0}), ("default", {})]
        with b.fb.tuning(mfma_rows=1):
            fits = [b.fb.fluxbin_plan_query(it["packs"][0], B)["kernel_name"] == "mfma_rows" for it in b.items]
        if any(fits):
            kernels.append(("mfma_rows", {"mfma_rows": 1}))
        runs = {k: [] for k, _ in kernels}
        for _ in range(rounds):
            for kern, tun in kernels:
                with b.fb.tuning(**tun):
                    for it in b.items:
                        it["ws"] = b.fb.make_workspace(it["packs"][0], B)
                    runs[kern].append(b.per_launch_us(launches, 3))
        us_k = {k: [statistics.median(v) for v in zip(*r)] for k, r in runs.items()}
        for i, it in enumerate(b.items):
            s = it["spec"]
            um, ul, us = us_k["mfma"][i], us_k["lut"][i], us_k["default"][i]
            plan = b.fb.fluxbin_plan_query(it["packs"][0], B)   # the launch plan's own choice (no forcing)
            row = {"us_per_call": round(us, 3), "GBps": round(it["bytes"] / (us * 1e-6) / 1e9, 1),
                   "tflop_eq": round(2.0 * B * s.M * (s.N + s.S) / (us * 1e-6) / 1e12, 2),
                   "matrix_core_kernel_us": round(um, 3), "lut_batch_kernel_us": round(ul, 3),
                   "default_kernel": plan["kernel_name"]}
            if "mfma_rows" in us_k and fits[i]:
                row["row_complete_matrix_core_kernel_us"] = round(us_k["mfma_rows"][i], 3)
            out[f"{s.name}_B{B}"] = row
        del b
        torch.cuda.empty_cache()
    return out


def prefill_us(specs, batches=(64, 256), launches=6):
    """Per-call microseconds at prefill-size batches: B > 32 runs as 32-row batch tiles (one launch each, every tile
    reading the packed weights again), graph-timed like the small-batch figures; TFLOP-eq counts 2 B M (N + S)."""
    import torch
    out = {}
    for B in batches:
        b = Bench(specs, B, COPIES_BYTES_PER_LAYER * len(specs))
        us = b.per_launch_us(launches, 3)
        for it, u in zip(b.items, us):
            s = it["spec"]
            plan = b.fb.fluxbin_plan_query(it["packs"][0], B)
            out[f"{s.name}_B{B}"] = {"us_per_call": round(u, 2), "us_per_batch_row": round(u / B, 3),
                                     "tflop_eq": round(2.0 * B * s.M * (s.N + s.S) / (u * 1e-6) / 1e12, 2),
                                     "batch_tiles": plan["batch_tiles"], "tile_kernel": plan["kernel_name"]}
        del b
        torch.cuda.empty_cache()
    return out


def decoder_layer_us(g_r: str, batches=(1, 4, 16), steps: int = 40):
    """A synthetic 70B decoder layer's linears in one HIP graph per step, for both hybrid variants (2 bases + 1%
    salient, 3 bases + 5% salient), at least three rotated copies of every layer; end-to-end microseconds per decoder
    layer and the whole layer's bytes per microsecond. Two launch sets: the seven linears (q, k, v, o, gate, up, down)
    and four fused launches (q|k|v stacked as one 10240-row layer, gate|up as one 57344-row layer, o, down)."""
    import torch
    from synth import config_layers, fused_decoder_layers
    out = {}
    allspecs = config_layers("c5_layer70b", g_r)
    fused = fused_decoder_layers(g_r)
    for variant in ("2b1pct", "3b5pct"):
        for kind, pool in (("", allspecs), ("_fused", fused)):
            specs = [sp for sp in pool if sp.name.startswith(variant)]
            b = Bench(specs, 1, 1.6e9, min_copies=3)
            for B in batches:
                if B != b.B:
                    b.set_batch(B)
                b.run(2, 2)   # warm up graph capture for this batch
                ms, _ = b.run(steps, 2, replays=5)
                us = sorted(ms)[len(ms) // 2] * 1000.0 / steps
                step_bytes = sum(it["bytes"] for it in b.items)
                out[f"{variant}{kind}_B{B}"] = {"us_per_layer": round(us, 2),
                                                "GBps": round(step_bytes / (us * 1e-6) / 1e9, 1),
                                                "calls": len(b.items),
                                                "copies_min": min(len(it["packs"]) for it in b.items)}
            del b
            torch.cuda.empty_cache()
    return out


def kernel_variants_us(g_r: str, launches: int = 40):
    """The 28672 x 8192 layer in the kernel variants the paper ablates (mu = 8 vs 4, pure global 3 and 4 bases, 2 bases
    + 1% salient), batch 1, graph-timed like the headline figure; the mu = 4 variant runs the generic kernel."""
    import torch
    from synth import kernel_variant_layers
    out = {}
    for spec in kernel_variant_layers(g_r):
        b = Bench([spec], 1, COPIES_BYTES_PER_LAYER)
        us = b.per_launch_us(launches, 3)[0]
        it = b.items[0]
        out[spec.name] = {"Kb": spec.Kb, "Ks": spec.Ks, "S": spec.S, "mu": spec.mu, "us_per_call": round(us, 3),
                          "bytes": it["bytes"], "GBps": round(it["bytes"] / (us * 1e-6) / 1e9, 1)}
        del b
        torch.cuda.empty_cache()
    return out


def small_layers_b1_us(g_r: str, launches: int = 60):
    """Batch 1 on the 7B attention (4096x4096) and MLP (11008x4096, 4096x11008) layers: the default launch plan's time,
    the split-tile kernel's (forced where the default is the row-complete kernel), and the stream probe, which issues
    the split-tile kernel's sign and row-scale requests without the table work (the load-only time of that access
    pattern on these small layers, start-up and end-of-grid included)."""
    import torch
    from synth import config_layers
    out = {}
    for cfg in ("c2_attn7b", "c3_mlp7b"):
        specs = config_layers(cfg, g_r)
        b = Bench(specs, 1, COPIES_BYTES_PER_LAYER * len(specs))
        kinds = [b.fb.fluxbin_plan_query(it["packs"][0], 1)["kernel_name"] for it in b.items]
        us = b.per_launch_us(launches, 3)
        with b.fb.tuning(rows=0):
            for it in b.items:
                it["ws"] = b.fb.make_workspace(it["packs"][0], 1)
            us_split = b.per_launch_us(launches, 3)
        probe = b.stream_probe_us(launches, 3)
        for it, kind, u, u2, pu in zip(b.items, kinds, us, us_split, probe):
            s = it["spec"]
            out[f"{cfg}_{s.name}"] = {"shape_out_x_in": f"{s.M}x{s.N}", "bytes": it["bytes"], "default_kernel": kind,
                                      "us_per_gemv": round(u, 3), "split_tile_kernel_us": round(u2, 3),
                                      "stream_probe_us": round(pu, 3), "us_over_probe": round(u / pu, 3),
                                      "GBps": round(it["bytes"] / (u * 1e-6) / 1e9, 1)}
        del b
        torch.cuda.empty_cache()
    return out


def shard_us(g_r: str, full_us: Dict[str, float], launches: int = 60):
    """One rank's share of the 70B MLP layers at P = 2, 4, 8 ranks (up split by output rows, down by input columns),
    batch 1: the kernel at the shard's real shape, against the full layer's time over P (what perfect splitting would
    give; the cross-rank sum of the down projection's partial outputs is not included)."""
    import torch
    from synth import shard_layers
    out = {}
    for P in (2, 4, 8):
        specs = shard_layers(P, g_r)
        b = Bench(specs, 1, COPIES_BYTES_PER_LAYER * len(specs))
        us = b.per_launch_us(launches, 3)
        for it, u, full in zip(b.items, us, ("up", "down")):
            s = it["spec"]
            out[s.name] = {"shape_out_x_in": f"{s.M}x{s.N}", "bytes": it["bytes"], "us_per_gemv": round(u, 3),
                           "GBps": round(it["bytes"] / (u * 1e-6) / 1e9, 1),
                           "pct_of_8TBps": round(100 * it["bytes"] / (u * 1e-6) / 1e9 / HBM_PEAK_GBS, 1),
                           "full_layer_us_over_P": round(full_us[full] / P, 3),
                           "kernel": b.fb.fluxbin_plan_query(it["packs"][0], 1)["kernel_name"]}
        del b
        torch.cuda.empty_cache()
    return out


def mu_profile_us(g_r: str, launches: int = 40):
    """mu = 8 against mu = 4 (same shapes and seeds) at batch 1 (Sec. 3.2 trades table size against lookups; App. E.2
    profiles mu on the 7B model): the 7B attention and MLP layers, the 70B MLP layers, and the distinct shapes of the
    70B decoder layer (q/o 8192x8192, k/v 1024x8192, gate/up 28672x8192, down 8192x28672) in both hybrid variants.
    The split-tile batch-1 kernel for both (its tables follow the packed mu); where the launch plan picks the
    row-complete kernel instead (its 16-entry tables serve either packing), that time is reported next to them."""
    import torch
    from synth import config_layers
    out = {}
    c5 = [sp for sp in config_layers("c5_layer70b", g_r) if sp.name.split("_", 1)[1] in ("q", "k", "gate", "down")]
    for cfg, specs in (("c2_attn7b", config_layers("c2_attn7b", g_r)), ("c3_mlp7b", config_layers("c3_mlp7b", g_r)),
                       ("c4_mlp70b", config_layers("c4_mlp70b", g_r)), ("c5_layer70b", c5)):
        for spec in specs:
            row = {"shape_out_x_in": f"{spec.M}x{spec.N}"}
            for mu in (8, 4):
                sp = spec.with_(mu=mu, name=f"{spec.name}_mu{mu}")
                b = Bench([sp], 1, COPIES_BYTES_PER_LAYER)
                it = b.items[0]
                if mu == 8 and b.fb.fluxbin_plan_query(it["packs"][0], 1)["kernel_name"] == "rows":
                    row["row_complete_kernel_us"] = round(b.per_launch_us(launches, 3)[0], 3)
                with b.fb.tuning(rows=0):
                    it["ws"] = b.fb.make_workspace(it["packs"][0], 1)
                    us = b.per_launch_us(launches, 3)[0]
                row[f"mu{mu}_us"] = round(us, 3)
                row[f"mu{mu}_GBps"] = round(it["bytes"] / (us * 1e-6) / 1e9, 1)
                del b
                torch.cuda.empty_cache()
            row["mu8_faster"] = row["mu8_us"] < row["mu4_us"]
            out[f"{cfg}_{spec.name}"] = row
    return out


# The paper's per-operator latencies on its NVIDIA A100 80GB (App. E.4, Table kernel-latency; batch 1, fp16
# activations, g = 128), in microseconds, by (out, in) shape and configuration: context for the MI355X figures.
PAPER_A100_KERNEL_US = {
    (4096, 4096): {"2b": 41, "2b-s8": 47, "2b-s16": 49, "4b": 56},
    (5120, 5120): {"2b": 63, "2b-s8": 73, "2b-s16": 74, "4b": 87},
    (4096, 11008): {"2b": 102, "2b-s8": 109, "2b-s16": 111, "4b": 158},
    (5120, 13824): {"2b": 167, "2b-s8": 166, "2b-s16": 169, "4b": 252},
}
# End-to-end decode speedup the paper quotes for LLaMA-2-7B 2b-s8-g128 against FP16 on that GPU (Sec. 4.1, Table
# llama2-task: 254.39 against 42.94 tokens/s).
PAPER_E2E_SPEEDUP = 5.92


def kernel_latency_grid_us(launches: int = 100):
    """The paper's kernel-latency table (App. E.4) on MI355X: four operator shapes x {2b, 2b-s8, 2b-s16, 4b}-g128
    (s8/s16: structured selection of s salient columns per 128, Ks = Kb = 2, one salient row scale per row and
    block), batch 1, graph-timed back-to-back launches over rotated packed copies (so every launch reads HBM), median of
    five replays. Next to each the paper's A100 latency, and per shape the cost of the salient refinement relative to
    the pure 2-base layer (the paper calls it nearly free)."""
    import torch
    from synth import kernel_latency_layers
    out = {}
    for spec in kernel_latency_layers():
        b = Bench([spec], 1, COPIES_BYTES_PER_LAYER)
        us = b.per_launch_us(launches, 5)[0]
        it = b.items[0]
        tag = spec.name.split("_", 1)[1].rsplit("-g", 1)[0]
        a100 = PAPER_A100_KERNEL_US[(spec.M, spec.N)][tag]
        out[spec.name] = {"us": round(us, 3), "bytes": it["bytes"], "GBps": round(it["bytes"] / (us * 1e-6) / 1e9, 1),
                          "pct_of_8TBps": round(100 * it["bytes"] / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 1),
                          "tflop_eq": round(2.0 * spec.M * (spec.N + spec.S) / (us * 1e-6) / 1e12, 2),
                          "kernel": b.fb.fluxbin_plan_query(it["packs"][0], 1)["kernel_name"],
                          "paper_A100_us": a100, "speedup_vs_paper_A100": round(a100 / us, 2)}
        del b
        torch.cuda.empty_cache()
    for (M, N) in PAPER_A100_KERNEL_US:
        base = out[f"{M}x{N}_2b-g128"]["us"]
        paper = PAPER_A100_KERNEL_US[(M, N)]
        for tag in ("2b-s8", "2b-s16"):
            out[f"{M}x{N}_{tag}_over_2b"] = {"mi355x": round(out[f"{M}x{N}_{tag}-g128"]["us"] / base, 3),
                                             "paper_A100": round(paper[tag] / paper["2b"], 3)}
    return out


def vcm_ablation_us(g_r: str, launches: int = 40):
    """The paper's VCM ablation on the 70B MLP layers: each layer as packed (salient columns repacked densely, VCM on)
    and as the same weights with the salient bases kept full width (VCM off: Ks more global bases with a column scale
    that is zero off the salient set), batch 1, graph-timed."""
    import torch
    from synth import config_layers, make_layer, vcm_off_equivalent
    out = {}
    for spec in config_layers("c4_mlp70b", g_r):
        L = make_layer(spec)
        for name, lay in (("vcm_on", L), ("vcm_off", vcm_off_equivalent(L))):
            b = Bench([lay.spec], 1, COPIES_BYTES_PER_LAYER, layers=[lay])
            us = b.per_launch_us(launches, 3)[0]
            it = b.items[0]
            out[f"{spec.name}_{name}"] = {"us_per_call": round(us, 3), "bytes": it["bytes"],
                                          "GBps": round(it["bytes"] / (us * 1e-6) / 1e9, 1)}
            del b
            torch.cuda.empty_cache()
    for nm in ("up", "down"):
        on, off = out[f"{nm}_vcm_on"]["us_per_call"], out[f"{nm}_vcm_off"]["us_per_call"]
        out[f"{nm}_latency_change_with_vcm"] = round(on / off - 1.0, 4)
    return out


def decomposition_ms(M: int = 8192, N: int = 8192, g: int = 128, s: int = 8, Kb: int = 2, Ks: int = 2, T: int = 10,
                     oracle_rows: int = 512):
    """The weight decomposition in the paper's 2b-s8-g128 configuration (Alg. FluxBin-Hybrid with a diagonal inverse
    Hessian: per g-column block the s most salient columns, Kb global bases, Ks salient bases of the block's residual
    on those columns, one row scale per row and block on both branches, T alternating rounds) of a synthetic M x N fp32
    matrix on the GPU (HIP events around the three library calls, median of 3), and the fp64 oracle on an
    oracle_rows x N slice of it on the host (one run), reported per million weights."""
    import numpy as np
    import torch
    from oracle import rc_oracle as rc
    from paper_2608_15602_amd import fluxbin as fb
    from synth import make_weight_matrix
    W, hinv = make_weight_matrix(M, N, seed=50, outlier_frac=0.01)
    Wt = torch.from_numpy(W).cuda()
    ht = torch.from_numpy(hinv).cuda()

    def run():
        _, _, mask = fb.fluxbin_structural_search(Wt, ht, g, s)
        gs, gar, gac = fb.fluxbin_rc_decompose(Wt, Kb, T, g)
        fb.fluxbin_rc_decompose(Wt, Ks, T, g, mask=mask, prior=(gs, gar, gac, g))

    run()
    torch.cuda.synchronize()
    ts = []
    for _ in range(3):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    gpu_ms = sorted(ts)[1]
    t0 = time.perf_counter()
    rc.hybrid_quantize(W[:oracle_rows].astype(np.float64), hinv, g=g, s=s, Kb=Kb, Ks=Ks, T=T)
    cpu_s = time.perf_counter() - t0
    return {"shape_out_x_in": f"{M}x{N}", "Kb": Kb, "Ks": Ks, "g": g, "s_per_group": s, "rounds": T,
            "gpu_ms": round(gpu_ms, 2), "gpu_ms_per_Mweight": round(gpu_ms / (M * N / 1e6), 4),
            "oracle_s_per_Mweight": round(cpu_s / (oracle_rows * N / 1e6), 4),
            "oracle_sample": f"rows 0..{oracle_rows - 1} (fp64 NumPy, {cpu_s:.1f} s)"}


def small_layer_us(spec, launches=200):
    """Per-call microseconds of a small layer (4096x4096): a HIP graph of back-to-back launches rotating distinct
    packed copies (so the signs come from HBM), median of 5 replays."""
    b = Bench([spec], 1, COPIES_BYTES_PER_LAYER)
    us = b.per_launch_us(launches, 5)[0]
    return us, b.items[0]["bytes"]


def summarize_trace(path: str, steps: int, warmup: int, replays: int) -> dict:
    """Split a rocprofv3 kernel trace (its kernel_trace.csv) of `bench.py --steps K --warmup W` into the run's phases:
    the batch-1 GEMV dispatches in launch order are W warmup steps (2 each), one graph upload replay (2K), then the
    `replays` timed replays (2K each); later dispatches belong to the per-layer figures. Returns the average dispatch
    duration of each phase and, for the timed replays, the median span from a replay's first dispatch start to its last
    dispatch end (compare with ms_per_step * K)."""
    import csv
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            if "k_gemv_b1" in r["Kernel_Name"]:
                rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    rows.sort()
    w, u, t = 2 * warmup, 2 * steps, 2 * steps * replays
    if len(rows) < w + u + t:
        raise SystemExit(f"trace has {len(rows)} GEMV dispatches, the headline phase needs {w + u + t}")
    avg = lambda seg: sum(e - s for s, e in seg) / len(seg) / 1e3
    timed = rows[w + u:w + u + t]
    spans = sorted((timed[k * u + u - 1][1] - timed[k * u][0]) / 1e6 for k in range(replays))
    return {"gemv_dispatches": len(rows), "warmup_avg_us": round(avg(rows[:w]), 3) if w else None,
            "upload_replay_avg_us": round(avg(rows[w:w + u]), 3), "timed_avg_us": round(avg(timed), 3),
            "timed_dispatches": t, "timed_replay_span_ms_median": round(spans[len(spans) // 2], 5),
            "later_avg_us": round(avg(rows[w + u + t:]), 3) if len(rows) > w + u + t else None}


def summarize_counters(path: str, launches: int, copy_bytes: int) -> dict:
    """One rocprofv3 counter pass (counter_collection.csv) of the counter-collection mode (`--copy-calib-mib`,
    `--eager-launches N`): the counter's value per dispatch (KiB) of the first three device-to-device copies of
    copy_bytes bytes (the calibration: bytes per counted KiB), and of the batch-1 GEMV dispatches, the first N the up
    layer and the next N the down layer; returns the calibrated bytes per launch of each layer."""
    import csv
    copies, gemv = [], []
    name = None
    with open(path) as f:
        for r in csv.DictReader(f):
            name = r["Counter_Name"]
            v = float(r["Counter_Value"])
            if "copyBuffer" in r["Kernel_Name"]:
                copies.append((int(r["Dispatch_Id"]), v))
            elif "k_gemv_b1" in r["Kernel_Name"]:
                gemv.append((int(r["Dispatch_Id"]), v))
    copies = [v for _, v in sorted(copies)][:3]
    gemv = [v for _, v in sorted(gemv)]
    if len(copies) < 3 or len(gemv) < 2 * launches:
        raise SystemExit(f"{path}: {len(copies)} copies and {len(gemv)} GEMV dispatches")
    cal = copy_bytes / (sum(copies) / len(copies))      # bytes per counted KiB
    mean = lambda xs: sum(xs) / len(xs)
    up, down = mean(gemv[:launches]), mean(gemv[launches:2 * launches])
    return {"counter": name, "copy_kib": round(mean(copies), 1), "bytes_per_counted_kib": round(cal, 3),
            "up_kib": round(up, 1), "down_kib": round(down, 1), "up_bytes": int(round(up * cal)),
            "down_bytes": int(round(down * cal))}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--replays", type=int, default=10, help="timed replays of the K-step graph (the median is reported)")
    ap.add_argument("--g-r", choices=["128", "N"], default="128")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-small", action="store_true", help="skip the 4096x4096 and small-batch per-call figures (70B and 7B MLP layers)")
    ap.add_argument("--no-decoder", action="store_true", help="skip the 70B decoder-layer graph figures")
    ap.add_argument("--no-variants", action="store_true", help="skip the kernel-variant figures (mu 4, pure global)")
    ap.add_argument("--no-grid", action="store_true", help="skip the paper's kernel-latency grid (App. E.4 shapes)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="before anything else, run a plain device-to-device copy of this many MiB three times "
                         "(the reference dispatch for HBM byte counters)")
    ap.add_argument("--eager-batch", type=int, default=1,
                    help="batch rows of the counter-collection launches (2..16: the small-batch product)")
    ap.add_argument("--eager-launches", type=int, default=0,
                    help="counter-collection mode: launch each layer this many times without graphs, then exit")
    ap.add_argument("--summarize-counters", metavar="COUNTER_COLLECTION_CSV",
                    help="no GPU work: calibrated bytes per launch of one rocprofv3 counter pass of the counter mode "
                         "(with the same --eager-launches and --copy-calib-mib)")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="no GPU work: split a rocprofv3 kernel trace of a run with the same --steps/--warmup/--replays "
                         "into its phases and print the batch-1 GEMV averages")
    args = ap.parse_args()
    if args.summarize_trace:
        print(json.dumps(summarize_trace(args.summarize_trace, args.steps, args.warmup, args.replays)))
        return
    if args.summarize_counters:
        print(json.dumps(summarize_counters(args.summarize_counters, args.eager_launches, args.copy_calib_mib << 20)))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU; sharding the path over several GPUs is not implemented",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from synth import config_layers
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    print(f"# device {torch.cuda.get_device_name(0)}", file=sys.stderr, flush=True)
    if args.copy_calib_mib > 0:
        n = args.copy_calib_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        print(f"# copy calibration: 3 x {n} bytes device-to-device", file=sys.stderr, flush=True)
    specs = config_layers("c4_mlp70b", args.g_r)
    bench = Bench(specs, 1, COPIES_BYTES_PER_LAYER * len(specs))
    print("# packed " + ", ".join(f"{it['spec'].name} x{len(it['packs'])}" for it in bench.items), file=sys.stderr,
          flush=True)
    if args.eager_launches > 0:
        if args.eager_batch != 1:
            bench.set_batch(args.eager_batch)
        for it in bench.items:
            for s in range(args.eager_launches):
                bench.launch(it, s)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "eager launches for counter collection", "launches_per_layer": args.eager_launches,
                          "batch": args.eager_batch,
                          "layers": [it["spec"].name for it in bench.items],
                          "bytes_per_launch": {it["spec"].name: it["bytes"] for it in bench.items}}), flush=True)
        return
    # Headline: a graph of exactly K steps (up then down per step, rotating packed copies), replayed `replays` times
    # back to back, each replay between HIP events on the replay stream; the median replay gives ms_per_step and value. Both launches
    # of a step are the batch-1 GEMV kernel, so its average launch duration in the timed region is the step time / 2
    # (gaps between the graph's launches included), and roofline.achieved comes from the same timing.
    replay_ms, wall = bench.run(args.steps, args.warmup, replays=args.replays)
    med_ms = sorted(replay_ms)[len(replay_ms) // 2]
    step_bytes = sum(it["bytes"] for it in bench.items)
    value = step_bytes * args.steps / (med_ms * 1e-3) / 1e9
    launch_us = med_ms * 1e3 / (args.steps * len(bench.items))
    achieved = (step_bytes / len(bench.items)) / (launch_us * 1e-6) / 1e9
    print(f"# headline: {args.replays} replays of {args.steps} steps, median {med_ms:.4f} ms", file=sys.stderr,
          flush=True)
    kern_us = bench.per_launch_us()
    probe_us = bench.stream_probe_us()
    cold_us = bench.cold_launch_us()
    traffic = measured_traffic()
    per_layer = {}
    for it, us, pus, cus in zip(bench.items, kern_us, probe_us, cold_us):
        s = it["spec"]
        per_layer[s.name] = {
            "shape_out_x_in": f"{s.M}x{s.N}", "us_per_gemv": round(us, 3),
            "GBps": round(it["bytes"] / (us * 1e-6) / 1e9, 1),
            "pct_of_8TBps": round(100 * it["bytes"] / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 1),
            "tflop_eq": round(2.0 * s.M * (s.N + s.S) / (us * 1e-6) / 1e12, 2),
            "bytes": it["bytes"], "lookups": it["lookups"],
            "stream_probe_us": round(pus, 3), "frac_of_stream_probe": round(pus / us, 4),
            "cold_single_launch_us": round(cus, 2),
        }
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(med_ms / args.steps, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded Llama-70B-shaped MLP layers; no trained weights)",
        "config": {"workload": WORKLOAD, "global_batch": 1, "g_r": args.g_r,
                   "timing": {"replays": args.replays, "replay_ms": [round(t, 4) for t in replay_ms],
                              "median_replay_ms": round(med_ms, 4), "us_per_launch": round(launch_us, 3)},
                   "layers": per_layer},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": (sum(traffic[it["spec"].name] for it in bench.items) // len(bench.items)
                                 if traffic else None),
                     "traffic_per_launch": traffic,
                     "kernel": "k_gemv_b1<8,1024,1,1,false> (both launches of a step); achieved = mean algorithmic "
                               "bytes per launch / (median replay time / launches per replay)",
                     "bytes_per_launch": {it["spec"].name: it["bytes"] for it in bench.items},
                     "frac_of_stream_probe": round(sum(probe_us) / sum(kern_us), 4)},
        "wall_s_timed": round(wall, 3),
    }
    if args.g_r == "128":   # the per-row reading (one row scale per row and base): 89.9 MB per 70B MLP layer
        bn = Bench(config_layers("c4_mlp70b", "N"), 1, COPIES_BYTES_PER_LAYER * 2)
        us_n = bn.per_launch_us()
        out["config"]["layers_g_r_N"] = {
            it["spec"].name: {"us_per_gemv": round(us, 3), "bytes": it["bytes"],
                              "GBps": round(it["bytes"] / (us * 1e-6) / 1e9, 1),
                              "pct_of_8TBps": round(100 * it["bytes"] / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 1)}
            for it, us in zip(bn.items, us_n)}
        del bn
        torch.cuda.empty_cache()
    if not args.no_small:
        spec2 = config_layers("c2_attn7b", args.g_r)[0]
        us, b2 = small_layer_us(spec2)
        out["config"]["attn_4096x4096_us_per_gemv"] = round(us, 3)
        out["config"]["attn_4096x4096_GBps"] = round(b2 / (us * 1e-6) / 1e9, 1)
        out["config"]["batch1_7b_layers"] = small_layers_b1_us(args.g_r)
        out["config"]["shards_mlp70b"] = shard_us(args.g_r, {it["spec"].name: u for it, u in zip(bench.items, kern_us)})
        out["config"]["small_batch"] = small_batch_us(specs, (2, 4, 8, 16))
        out["config"]["small_batch_mlp7b"] = small_batch_us(config_layers("c3_mlp7b", args.g_r), (2, 4, 8))
        out["config"]["small_batch_attn7b"] = small_batch_us(config_layers("c2_attn7b", args.g_r), (2, 4, 8))
        out["config"]["prefill_mlp70b"] = prefill_us(specs)
    if not args.no_grid:
        out["config"]["kernel_latency_grid"] = kernel_latency_grid_us()
    if not args.no_decoder:
        out["config"]["decoder_layer_70b"] = decoder_layer_us(args.g_r)
    if not args.no_variants:
        out["config"]["kernel_variants_28672x8192"] = kernel_variants_us(args.g_r)
        out["config"]["vcm_ablation"] = vcm_ablation_us(args.g_r)
        out["config"]["mu_profile"] = mu_profile_us(args.g_r)
        out["config"]["decomposition"] = decomposition_ms()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(bench, args.cpu_budget)
    # Context only (another GPU, and an end-to-end figure): the paper's own numbers next to this run's.
    ctx = {"paper_hardware": "NVIDIA A100 80GB",
           "paper_e2e_decode_speedup_vs_fp16": PAPER_E2E_SPEEDUP,
           "paper_e2e_note": "LLaMA-2-7B 2b-s8-g128 against FP16, end to end (Sec. 4.1); not a kernel figure",
           "paper_a100_kernel_us": {f"{M}x{N}": v for (M, N), v in PAPER_A100_KERNEL_US.items()}}
    if "cpu_baseline" in out and out["cpu_baseline"].get("value"):
        ctx["gpu_over_cpu_oracle"] = round(value / out["cpu_baseline"]["value"], 1)
        ctx["gpu_over_cpu_oracle_note"] = "the oracle is an untuned fp64 correctness reference, not a CPU kernel"
    out["paper_context"] = ctx
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
