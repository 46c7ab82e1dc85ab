"""Benchmark: one decode step of the 35B-class int4 MoE layer at batch 1.

A step is the whole hot path on one token: layer input (RMSNorm -> fp16),
router + softmax-top-k, prerouter prediction for the next layer, the 8
routed + 1 shared int4 group-64 SwiGLU experts with the unmerged LoRA delta,
and the combine.  Steps rotate over 32 resident layer instances (32 x ~520 MB)
so that weights come from HBM and not from the 256 MB last-level cache.  The
K timed steps are replayed from one captured HIP graph, inputs resident in
HBM.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, published
METRIC = "int4 MoE layer achieved HBM GB/s (% peak) at batch 1; tokens/s, 40-layer stack"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def proj_bytes(out_dim, in_dim):
    """Stored bytes of an int4 g64 projection: codes + one (fp16 s, fp16 z) per 64."""
    return out_dim * in_dim // 2 + out_dim * (in_dim // 64) * 4


def layer_bytes(wl):
    """Algorithmic bytes of one decode step: the weights the method must read
    once per token (selected experts + shared, their LoRA, router, head) plus
    the token's input and output vectors."""
    n = wl.K + wl.S
    expert = 2 * proj_bytes(wl.I, wl.d) + proj_bytes(wl.d, wl.I)
    lora = 2 * (2 * (wl.r * wl.d + wl.I * wl.r) + wl.r * wl.I + wl.d * wl.r)
    ffn = n * (expert + lora)
    route = 2 * wl.E * wl.d * 2                    # router + prerouter head, fp16
    io = wl.d * 4 + wl.d * 2 + wl.d * 4            # xi read, x write, y write
    # dominant kernel (gate/up stage): gate + up codes, scales/zeros, LoRA A, and x
    gateup = n * (2 * proj_bytes(wl.I, wl.d) + 2 * wl.r * wl.d * 2) + wl.d * 2
    return {"ffn": ffn, "route": route, "io": io, "step": ffn + route + io, "gateup": gateup}


class Hip:
    """The few HIP runtime calls the benchmark makes itself (event timing)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        assert self.lib.hipEventCreate(ctypes.byref(e)) == 0
        return e.value

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        assert self.lib.hipEventSynchronize(ctypes.c_void_p(b)) == 0
        assert self.lib.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a),
                                            ctypes.c_void_p(b)) == 0
        return ms.value

    def destroy(self, e):
        self.lib.hipEventDestroy(ctypes.c_void_p(e))


def build_instances(wl, n_inst, torch):
    """n_inst copies of one seeded layer (all 256 + 1 experts, router, head)
    at distinct device addresses, bound in one slot table (one table layer
    per instance, a seeded slot permutation)."""
    import synth
    from paper_2609_18063_amd import binding as B, weights as W
    t0 = time.time()
    n_ids = wl.E + wl.S
    bundles = [synth.bundle(wl, 0, e) for e in range(n_ids)]
    router = synth.router_weights(wl, 0, 0)
    head = synth.router_weights(wl, 0, 1)
    buf, boffs, eoffs = W.pack_host(bundles, extra=[router, head])
    log("packed one layer instance: %.1f MB in %.1fs" % (buf.nbytes / 1e6, time.time() - t0))
    host = torch.from_numpy(buf).pin_memory()
    table = B.SlotTable(n_inst, n_ids, n_ids)
    perm = np.random.default_rng(1000).permutation(n_ids)
    inst = []
    for i in range(n_inst):
        dev = torch.empty(buf.nbytes, dtype=torch.uint8, device="cuda")
        dev.copy_(host, non_blocking=True)
        W.bind_layer(table, i, dev, boffs, perm)
        inst.append({
            "dev": dev,
            "router": W.extra_tensor(dev, eoffs[0], router.shape, torch.float16),
            "head": W.extra_tensor(dev, eoffs[1], head.shape, torch.float16),
        })
    table.sync()
    torch.cuda.synchronize()
    log("uploaded %d instances (%.1f GB) in %.1fs" % (n_inst, n_inst * buf.nbytes / 1e9,
                                                        time.time() - t0))
    return table, inst


def step(B, spec, table, inst, i, xi_row, bufs):
    """Enqueue one decode step of instance ``i`` on the current stream."""
    B.rmsnorm_f16(xi_row, bufs["x"])
    B.route(spec, bufs["x"], inst["router"], bufs["idx"], bufs["w"], bufs["ws"])
    B.preroute(spec, bufs["x"], inst["head"], bufs["pidx"], bufs["pw"], bufs["ws"])
    B.expert_ffn(spec, table, i, bufs["x"], bufs["idx"], bufs["ye"], bufs["status"], bufs["ws"])
    B.combine(spec, bufs["ye"], bufs["w"], bufs["y"])


def cpu_baseline(wl, budget_s=15.0):
    """The oracle as it stands, on a bounded sample of the same workload."""
    import synth
    from oracle import expert as o_expert, routing as o_routing
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    router = synth.router_weights(wl, 0, 0)
    head = synth.router_weights(wl, 0, 1)
    shared = [synth.bundle(wl, 0, wl.E + s) for s in range(wl.S)]
    cache = {}
    done, spent = 0, 0.0
    while spent < budget_s and done < 200:
        xi = synth.token_draws(wl, done, 1)[0]
        x16 = o_routing.rms_norm_f16(xi)
        _, inds, _ = o_routing.route(router, x16, wl.K)
        for e in inds:                      # inputs are prepared outside the timed region
            if int(e) not in cache:
                cache[int(e)] = synth.bundle(wl, 0, int(e))
        t0 = time.perf_counter()
        o_routing.rms_norm_f16(xi)
        o_expert.moe_layer(x16, wl.K, lambda e: cache[e], shared, wl.lora_scale,
                           w_router16=router, w_head16=head)
        spent += time.perf_counter() - t0
        done += 1
    per_tok = spent / done
    return {"value": round(layer_bytes(wl)["step"] / per_tok / 1e9, 4), "unit": "GB/s",
            "cores": int(threads), "kind": "oracle",
            "sample": "%d tokens of the 35B-class layer (float64 oracle, %.2f s/token)"
                      % (done, per_tok)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--instances", type=int, default=32)
    ap.add_argument("--prof-launches", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only; a multi-GPU (expert-parallel) run is not "
              "implemented.", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2609_18063_amd import binding as B

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    B.lib()
    wl = synth.WORKLOADS["moe35b"]
    spec = B.spec_from_workload(wl)
    nb = layer_bytes(wl)
    K, W = args.steps, args.warmup
    table, inst = build_instances(wl, args.instances, torch)

    tokens = torch.from_numpy(synth.token_draws(wl, 0, K + W)).cuda()
    n = wl.K + wl.S
    bufs = {
        "ws": torch.zeros(B.workspace_bytes(spec, 1), dtype=torch.uint8, device="cuda"),
        "x": torch.empty(1, wl.d, dtype=torch.float16, device="cuda"),
        "idx": torch.empty(1, wl.K, dtype=torch.int32, device="cuda"),
        "w": torch.empty(1, wl.K, dtype=torch.float32, device="cuda"),
        "pidx": torch.empty(1, wl.K, dtype=torch.int32, device="cuda"),
        "pw": torch.empty(1, wl.K, dtype=torch.float32, device="cuda"),
        "ye": torch.empty(1, n, wl.d, dtype=torch.float32, device="cuda"),
        "y": torch.empty(1, wl.d, dtype=torch.float32, device="cuda"),
        "status": torch.zeros(1, dtype=torch.int32, device="cuda"),
    }
    # eager run once to load kernels, then capture warmup and timed graphs
    step(B, spec, table, inst[0], 0, tokens[0:1], bufs)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    graphs = {}
    for name, t0, count in (("warmup", K, W), ("timed", 0, K)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for j in range(count):
                i = (t0 + j) % args.instances
                step(B, spec, table, inst[i], i, tokens[t0 + j:t0 + j + 1], bufs)
        graphs[name] = g
    torch.cuda.synchronize()
    log("captured graphs: %d warmup + %d timed steps" % (W, K))

    if W:
        graphs["warmup"].replay()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    ev0.record()
    graphs["timed"].replay()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / K
    assert int(bufs["status"].item()) == 0, "slot miss or bad index during the benchmark"
    gbs = nb["step"] * K / (ms_total * 1e-3) / 1e9
    log("timed %d steps: %.3f ms GPU (%.3f ms wall), %.2f us/step, %.1f GB/s"
        % (K, ms_total, wall * 1e3, ms_step * 1e3, gbs))

    # per-launch duration of the dominant kernel (gate/up expert stage)
    hip = Hip()
    evs = [(hip.event(), hip.event()) for _ in range(args.prof_launches)]
    for j, (a, b) in enumerate(evs):
        i = j % args.instances
        B.profile_arm(B.MOE_PROF_FFN_MAIN, a, b)
        B.expert_ffn(spec, table, i, bufs["x"], bufs["idx"], bufs["ye"], bufs["status"], bufs["ws"])
    torch.cuda.synchronize()
    durs = [hip.elapsed_ms(a, b) for a, b in evs]
    for a, b in evs:
        hip.destroy(a)
        hip.destroy(b)
    dom_ms = float(np.mean(durs))
    achieved = nb["gateup"] / (dom_ms * 1e-3) / 1e9
    log("gate/up kernel: mean %.2f us, median %.2f us over %d launches -> %.1f GB/s"
        % (dom_ms * 1e3, float(np.median(durs)) * 1e3, len(durs), achieved))

    cpu = None if args.no_cpu_baseline else cpu_baseline(wl)
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded int4 g64 experts, fp16 LoRA / router / head, N(0,1) tokens)",
        "config": {
            "workload": "moe35b decode layer at batch 1: d 2048, 256 experts top-8 + 1 shared, "
                        "I 512, int4 g64 + fp16 (s,z), LoRA r16 on gate/up/down, router + "
                        "prerouter fp16 [256x2048]; %d rotated layer instances" % args.instances,
            "tokens": K,
            "bytes_per_step": nb["step"],
        },
        "pct_peak_hbm": round(100.0 * gbs / PEAK_HBM_GBS, 2),
        "roofline": {
            "bound": "hbm",
            "kernel": "ffn_gateup_kernel (gate/up int4 matvecs + LoRA A)",
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": None,
            "bytes_per_launch": nb["gateup"],
            "mean_launch_us": round(dom_ms * 1e3, 3),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
