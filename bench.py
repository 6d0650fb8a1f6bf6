"""Benchmark of the D^2MoE MoE-layer hot path on one MI355X.

Workload: a Mixtral-8x7B-shaped MoE layer in decode (d_model 4096, d_ff 14336,
8 SwiGLU experts, top-2), a batch of 16 tokens, one request per token, each
(request, expert) bit-width drawn from {2,3,4,8} with probabilities
{.2,.3,.3,.2}; weights N(0, 0.02) MWQ-packed with group 128 and an 8-bit nest;
bf16 activations N(0,1).  Eight independently drawn layers rotate from step to
step so that the weight reads miss the 256 MB last-level cache.  A step is one
layer call: route (gate, top-k, bit lookup, histogram/permutation) plus the
expert forward (W1/W3 + SwiGLU, W2, combine).

Prints one JSON line.  `value` = tokens per second of the whole step with
inputs resident in HBM, timed over replays of one captured HIP graph per
layer step (route + forward, as a serving loop would launch it; --eager times
eager launches instead; the eager step time is always reported as
ms_per_step_eager);
`roofline` = algorithmic bytes of the dominant kernel (W1/W3 expert kernel:
packed planes, scales and zeros of every active expert up to its largest
requested bit-width) per launch over its average duration, timed with HIP
events on the stream it runs on during the eager pass; `cpu_baseline` = the
CPU oracle on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("MoE-layer tokens/s + achieved HBM GB/s (fraction of peak) at mixed 2/3/4/8-bit "
          "experts")
HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


# The GPU leaves its idle clocks only after some milliseconds of sustained
# load: at the Mixtral decode step the first 16 steps averaged 0.64 ms, steps
# 16-31 0.31 ms, 32-47 0.28 ms, and every later block of 16 0.261-0.268 ms.
# Every timed workload is therefore preceded by its warm-up steps and then by
# more untimed steps until the GPU has been kept busy for WARM_MS.
WARM_MS = 100.0


def warm(step, warmup, min_ms=WARM_MS):
    """Untimed warm-up: `warmup` calls of step(i), then further calls in
    batches of 16 until at least min_ms of wall time has passed with the GPU
    busy.  Returns the number of calls made (the next step index)."""
    import torch
    n = 0
    for _ in range(warmup):
        step(n)
        n += 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < min_ms:
        for _ in range(16):
            step(n)
            n += 1
        torch.cuda.synchronize()
    return n


def mwq_bytes(rows, cols, group, b_min, bits):
    """Packed bytes of a b-bit read of one [rows][cols] matrix: b planes,
    the scales of levels <= b and the zeros."""
    if bits <= 0:
        return 0
    ng = cols // group
    return rows * cols * bits // 8 + rows * ng * 2 * (bits - b_min + 1) + rows * ng


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batch", type=int, default=16)
    ap.add_argument("--layers", type=int, default=8)
    ap.add_argument("--sweep", default="1,4",
                    help="extra batch sizes of the same decode layer reported alongside")
    ap.add_argument("--tiny-steps", type=int, default=100,
                    help="also time the tiny layer (d_model 256, d_ff 512, 8 experts top-2, "
                         "64 fp32 tokens; 0: skip)")
    ap.add_argument("--no-calib", dest="calib", action="store_false",
                    help="skip timing the calibration-aware MWQ setup (factor and calibrated "
                         "pack of one Mixtral W1/W3 and W2 expert)")
    ap.add_argument("--stream-steps", type=int, default=3,
                    help="also time the Mixtral decode layer with its experts streamed from "
                         "pinned host memory, HEBF against ascending unit order (0: skip)")
    ap.add_argument("--ceiling-gib", type=float, default=4.0,
                    help="size of the plain streaming read that measures this GPU's HBM read "
                         "ceiling in the same run (0: skip)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--prefill-steps", type=int, default=5,
                    help="also time the 2048-token prefill of the same layers (0: skip)")
    ap.add_argument("--fine-steps", type=int, default=10,
                    help="also time the 512-token fine-grained layer (64 routed experts top-6 "
                         "plus a shared expert; 0: skip)")
    ap.add_argument("--stack-steps", type=int, default=128,
                    help="also run the 32-layer decoder stack of MoE layers, 64 sequences, "
                         "this many decode steps (0: skip)")
    ap.add_argument("--variant-steps", type=int, default=40,
                    help="also time batch-16 decode under the paper's two nests (b 2-4, b 5-8) "
                         "and the LLaMA2-13B-shaped dense FFN (0: skip)")
    ap.add_argument("--no-learned", dest="learned", action="store_false",
                    help="skip the decode step with learned bit-width routers")
    ap.add_argument("--eager", dest="graph", action="store_false",
                    help="time eager launches instead of replays of one captured HIP graph per "
                         "layer step (the eager step time is reported either way)")
    ap.add_argument("--dump-steps", action="store_true",
                    help="print the per-step times of the main workload to stderr")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 256 MiB device copy three times (reference for "
                         "hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library runs the MoE layer on a single "
              "MI355X and has no multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2504_15299_amd import api

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    d, f, E, k, g, b_min, b_max = 4096, 14336, 8, 2, 128, 2, 8
    use_graphs = args.graph
    NL = args.layers

    # ---- resident packed weights, one set per rotating layer ----
    t0 = time.time()
    gen = torch.Generator(device=dev)
    layers = []
    for l in range(NL):
        w13 = api.MWQ.empty(E, 2 * f, d, g, b_min, b_max, device=dev)
        w2 = api.MWQ.empty(E, d, f, g, b_min, b_max, device=dev)
        for e in range(E):
            gen.manual_seed(1_000_003 * l + 2 * e)
            W = torch.randn((1, 2 * f, d), generator=gen, device=dev) * 0.02
            api.pack_mwq(W, w13.expert(e))
            gen.manual_seed(1_000_003 * l + 2 * e + 1)
            W = torch.randn((1, d, f), generator=gen, device=dev) * 0.02
            api.pack_mwq(W, w2.expert(e))
            del W
        gen.manual_seed(7_000_000 + l)
        Wg = torch.randn((E, d), generator=gen, device=dev) * 0.02
        layers.append((w13, w2, Wg))
    torch.cuda.synchronize()
    pack_s = time.time() - t0

    def run_batch(T, steps, warmup, profile):
        rng = np.random.default_rng(2 + T)
        x = torch.from_numpy(rng.standard_normal((T, d), dtype=np.float32)).to(dev).to(torch.bfloat16)
        req = torch.arange(T, dtype=torch.int32, device=dev)
        tables = [torch.from_numpy(rng.choice(np.array([2, 3, 4, 8], np.uint8), size=(T, E),
                                              p=[0.2, 0.3, 0.3, 0.2])).to(dev)
                  for _ in range(NL)]
        routs = [api.Routing.empty(T, E, k, b_min, b_max, device=dev) for _ in range(NL)]
        out = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, d, f, E, k), dtype=torch.uint8, device=dev)

        def step(i, events=None):
            l = i % NL
            w13, w2, Wg = layers[l]
            api.route(x, Wg, None, k, req, tables[l], b_min, b_max, out=routs[l])
            api.moe_forward(x, w13, w2, routs[l], k, out=out, workspace=ws, events=events)

        w0 = warm(step, warmup)
        # eager pass: per-kernel durations from HIP events on the launch stream
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        for row in evs:            # torch creates the HIP event at its first record
            for ev in row:
                ev.record()
        torch.cuda.synchronize()
        # one stream marker at every step boundary: per-step durations
        bounds = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        for ev in bounds:
            ev.record()
        torch.cuda.synchronize()
        t_start, t_stop = bounds[0], bounds[-1]
        t_start.record()
        for i in range(steps):
            step(w0 + i, evs[i] if profile else None)
            bounds[i + 1].record()
        torch.cuda.synchronize()
        ms_eager = t_start.elapsed_time(t_stop) / steps
        per_step = np.array([bounds[i].elapsed_time(bounds[i + 1]) for i in range(steps)])
        ms = ms_eager
        if use_graphs:
            # one captured step (route + forward) per rotating layer, replayed
            cur = torch.cuda.current_stream()
            side = torch.cuda.Stream()
            side.wait_stream(cur)
            with torch.cuda.stream(side):
                for l in range(NL):
                    step(l)
            cur.wait_stream(side)
            torch.cuda.synchronize()
            graphs = []
            for l in range(NL):
                g_ = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g_):
                    step(l)
                graphs.append(g_)
            wg = warm(lambda i: graphs[i % NL].replay(), warmup)
            t_start.record()
            for i in range(steps):
                graphs[(wg + i) % NL].replay()
            t_stop.record()
            torch.cuda.synchronize()
            ms = t_start.elapsed_time(t_stop) / steps
        # algorithmic bytes per layer call from each layer's routing
        alg13, alg2 = [], []
        for l in range(NL):
            mb = routs[l].expert_maxbit.cpu().numpy()
            alg13.append(sum(mwq_bytes(2 * f, d, g, b_min, int(b)) for b in mb))
            alg2.append(sum(mwq_bytes(d, f, g, b_min, int(b)) for b in mb))
        per_step13 = [alg13[(w0 + i) % NL] for i in range(steps)]
        per_step2 = [alg2[(w0 + i) % NL] for i in range(steps)]
        res = dict(T=T, warmup_steps_run=w0, ms_per_step=ms, ms_per_step_eager=ms_eager,
                   tokens_per_s=T / (ms * 1e-3),
                   layer_bytes=float(np.mean([a + b for a, b in zip(per_step13, per_step2)])))
        res["layer_GBps"] = res["layer_bytes"] / (ms * 1e-3) / 1e9
        res["step_ms_p10_p50_p90"] = [round(float(v), 5) for v in
                                      np.percentile(per_step, [10, 50, 90])]
        res["per_step_ms"] = [round(float(v), 4) for v in per_step]
        if profile:
            d13 = np.array([e[0].elapsed_time(e[1]) for e in evs])
            res["w13_ms_p10_p50_p90"] = [round(float(v), 5) for v in np.percentile(d13, [10, 50, 90])]
            res["per_step_w13_ms"] = [round(float(v), 4) for v in d13]
            d2 = np.array([e[2].elapsed_time(e[3]) for e in evs])
            res["w13_ms"] = float(d13.mean())
            res["w2_ms"] = float(d2.mean())
            res["w13_GBps"] = float(np.mean(per_step13) / (d13.mean() * 1e-3) / 1e9)
            res["w2_GBps"] = float(np.mean(per_step2) / (d2.mean() * 1e-3) / 1e9)
            res["w13_bytes"] = float(np.mean(per_step13))
        return res

    def run_prefill(steps, warmup):
        """Prefill of the same layers: 2048 tokens from 4 requests of 512,
        per-request bit tables from {2,4,8}, gate bias ln p_e with
        p_e ~ (e+1)^-1.1 so that expert load follows Zipf(1.1).  Returns the
        step time and the expert GEMMs' rate in algorithmic TFLOP/s
        (2 * 3 * d * d_ff per routed token, the W1/W3 and W2 kernels timed
        with HIP events)."""
        T, R = 2048, 4
        rng = np.random.default_rng(3)
        x = torch.from_numpy(rng.standard_normal((T, d), dtype=np.float32)).to(dev).to(torch.bfloat16)
        req = torch.from_numpy((np.arange(T) // (T // R)).astype(np.int32)).to(dev)
        p = (np.arange(E) + 1.0) ** -1.1
        bias = torch.from_numpy(np.log(p / p.sum()).astype(np.float32)).to(dev)
        tables = [torch.from_numpy(rng.choice(np.array([2, 4, 8], np.uint8), size=(R, E))).to(dev)
                  for _ in range(NL)]
        routs = [api.Routing.empty(T, E, k, b_min, b_max, device=dev) for _ in range(NL)]
        out = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, d, f, E, k), dtype=torch.uint8, device=dev)

        def step(i, events=None):
            l = i % NL
            w13, w2, Wg = layers[l]
            api.route(x, Wg, bias, k, req, tables[l], b_min, b_max, out=routs[l])
            api.moe_forward(x, w13, w2, routs[l], k, out=out, workspace=ws, events=events)

        w0 = warm(step, warmup)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        for row in evs:
            for ev in row:
                ev.record()
        torch.cuda.synchronize()
        t_start = torch.cuda.Event(enable_timing=True)
        t_stop = torch.cuda.Event(enable_timing=True)
        t_start.record()
        for i in range(steps):
            step(w0 + i, evs[i])
        t_stop.record()
        torch.cuda.synchronize()
        ms = t_start.elapsed_time(t_stop) / steps
        ms_eager = ms
        if use_graphs:
            # the kernel times above come from the eager steps' events; the
            # step time from replays of one captured step per layer
            cur = torch.cuda.current_stream()
            side = torch.cuda.Stream()
            side.wait_stream(cur)
            with torch.cuda.stream(side):
                for l in range(NL):
                    step(l)
            cur.wait_stream(side)
            torch.cuda.synchronize()
            graphs = []
            for l in range(NL):
                g_ = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g_):
                    step(l)
                graphs.append(g_)
            wg = warm(lambda i: graphs[i % NL].replay(), warmup)
            t_start.record()
            for i in range(steps):
                graphs[(wg + i) % NL].replay()
            t_stop.record()
            torch.cuda.synchronize()
            ms = t_start.elapsed_time(t_stop) / steps
        d13 = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
        d2 = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
        flop13 = 2.0 * 2 * d * f * T * k
        flop2 = 2.0 * d * f * T * k
        hist = routs[(w0 + steps - 1) % NL].hist.cpu().numpy().sum(axis=1)
        return {"tokens": T, "ms_per_step": round(ms, 4), "ms_per_step_eager": round(ms_eager, 4),
                "launch": "hip graph per layer step" if use_graphs else "eager",
                "tokens_per_s": round(T / (ms * 1e-3), 1),
                "w13_ms": round(d13, 4), "w2_ms": round(d2, 4),
                "w13_TFLOPs": round(flop13 / (d13 * 1e-3) / 1e12, 1),
                "w2_TFLOPs": round(flop2 / (d2 * 1e-3) / 1e12, 1),
                "expert_TFLOPs": round((flop13 + flop2) / ((d13 + d2) * 1e-3) / 1e12, 1),
                "mfma_peak_TFLOPs": MFMA_BF16_PEAK_TFLOPS,
                "mfma_frac": round((flop13 + flop2) / ((d13 + d2) * 1e-3) / 1e12
                                   / MFMA_BF16_PEAK_TFLOPS, 4),
                "expert_load": [int(v) for v in hist]}

    def run_fine(steps, warmup, copies=4):
        """Fine-grained MoE layer: d_model 2048, 64 routed SwiGLU experts d_ff
        1408 (top-6) plus one shared expert d_ff 5632 at 8 bits, 512 tokens,
        MWQ group 64 nested to 8 bits.  Bit-widths hottest-first: a first
        routing pass (untimed) counts each expert's tokens; the 16 most routed
        get 8 bits, the next 16 get 4, the next 16 get 3, the rest 2.  Four
        independently drawn copies rotate.  Reports tokens/s, the algorithmic
        HBM bytes (active experts at their largest bit-width plus the shared
        expert) and flops of the step, and both roofline fractions."""
        dF, fF, EF, kF, gF, fS, T = 2048, 1408, 64, 6, 64, 5632, 512
        rng = np.random.default_rng(4)
        x = torch.from_numpy(rng.standard_normal((T, dF), dtype=np.float32)).to(dev).to(torch.bfloat16)
        sets = []
        for c in range(copies):
            w13 = api.MWQ.empty(EF, 2 * fF, dF, gF, b_min, b_max, device=dev)
            w2 = api.MWQ.empty(EF, dF, fF, gF, b_min, b_max, device=dev)
            gen.manual_seed(9_000_000 + c)
            api.pack_mwq(torch.randn((EF, 2 * fF, dF), generator=gen, device=dev) * 0.02, w13)
            api.pack_mwq(torch.randn((EF, dF, fF), generator=gen, device=dev) * 0.02, w2)
            s13 = api.MWQ.empty(1, 2 * fS, dF, gF, b_min, b_max, device=dev)
            s2 = api.MWQ.empty(1, dF, fS, gF, b_min, b_max, device=dev)
            api.pack_mwq(torch.randn((1, 2 * fS, dF), generator=gen, device=dev) * 0.02, s13)
            api.pack_mwq(torch.randn((1, dF, fS), generator=gen, device=dev) * 0.02, s2)
            Wg = torch.randn((EF, dF), generator=gen, device=dev) * 0.02
            probe = api.route(x, Wg, None, kF, None, torch.full((1, EF), 8, dtype=torch.uint8,
                                                               device=dev), b_min, b_max)
            counts = probe.hist.sum(dim=1).cpu().numpy()
            order = sorted(range(EF), key=lambda e: (-int(counts[e]), e))
            tb = np.full((1, EF), 2, np.uint8)
            for rank, e in enumerate(order[:48]):
                tb[0, e] = (8, 4, 3)[rank // 16]
            table = torch.from_numpy(tb).to(dev)
            r = api.Routing.empty(T, EF, kF, b_min, b_max, device=dev)
            sets.append((w13, w2, s13, s2, Wg, table, r))
            torch.cuda.synchronize()
        out = torch.empty((T, dF), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, dF, fF, EF, kF, shared_d_ff=fS),
                         dtype=torch.uint8, device=dev)

        def step(i):
            w13, w2, s13, s2, Wg, table, r = sets[i % copies]
            api.route(x, Wg, None, kF, None, table, b_min, b_max, out=r)
            api.moe_forward(x, w13, w2, r, kF, shared=(s13, s2, 8), out=out, workspace=ws)

        w0 = warm(step, warmup)
        t_start = torch.cuda.Event(enable_timing=True)
        t_stop = torch.cuda.Event(enable_timing=True)
        t_start.record()
        for i in range(steps):
            step(w0 + i)
        t_stop.record()
        torch.cuda.synchronize()
        ms = t_start.elapsed_time(t_stop) / steps
        ms_eager = ms
        if use_graphs:
            # one captured step (route + forward) per copy, replayed
            cur = torch.cuda.current_stream()
            side = torch.cuda.Stream()
            side.wait_stream(cur)
            with torch.cuda.stream(side):
                for c in range(copies):
                    step(c)
            cur.wait_stream(side)
            torch.cuda.synchronize()
            graphs = []
            for c in range(copies):
                g_ = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g_):
                    step(c)
                graphs.append(g_)
            wg = warm(lambda i: graphs[i % copies].replay(), warmup)
            w0 = wg
            t_start.record()
            for i in range(steps):
                graphs[(wg + i) % copies].replay()
            t_stop.record()
            torch.cuda.synchronize()
            ms = t_start.elapsed_time(t_stop) / steps
        byts = []
        for c in range(copies):
            mb = sets[c][6].expert_maxbit.cpu().numpy()
            byts.append(sum(mwq_bytes(2 * fF, dF, gF, b_min, int(b)) + mwq_bytes(dF, fF, gF, b_min, int(b))
                            for b in mb)
                        + mwq_bytes(2 * fS, dF, gF, b_min, 8) + mwq_bytes(dF, fS, gF, b_min, 8))
        nbytes = float(np.mean([byts[(w0 + i) % copies] for i in range(steps)]))
        flop = 2.0 * 3 * dF * fF * T * kF + 2.0 * 3 * dF * fS * T
        gbps = nbytes / (ms * 1e-3) / 1e9
        tflops = flop / (ms * 1e-3) / 1e12
        return {"workload": "fine-grained MoE layer (d_model 2048, 64 routed SwiGLU experts "
                            "d_ff 1408 top-6, shared expert d_ff 5632 at 8 bits, 512 tokens, "
                            "group 64, bits hottest-first 8/4/3/2), 4 rotating copies",
                "tokens": T, "ms_per_step": round(ms, 4), "ms_per_step_eager": round(ms_eager, 4),
                "launch": "hip graph per step" if use_graphs else "eager",
                "tokens_per_s": round(T / (ms * 1e-3), 1), "alg_bytes": nbytes, "hbm_GBps": round(gbps, 1),
                "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "alg_GFLOP": round(flop / 1e9, 2),
                "TFLOPs": round(tflops, 1), "mfma_frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4)}

    def run_stack(steps, n_layers=32, T=64, eps=1e-5):
        """Decoder stack: n_layers Mixtral-8x7B-shaped MoE layers, each block
        x <- x + MoE_l(rmsnorm(x)) (attention absent), all layers resident,
        MWQ group 128 nested to 8 bits; 64 sequences, each a request with one
        bit-width tier from {2,4,8} for every expert and layer; each decode
        step feeds the previous step's final hidden state.  Reports tokens/s
        over all steps and the algorithmic HBM bytes of a step (every layer's
        active experts at their largest bit-width, from the last step's
        routing)."""
        stack = []
        for l in range(n_layers):
            w13 = api.MWQ.empty(E, 2 * f, d, g, b_min, b_max, device=dev)
            w2 = api.MWQ.empty(E, d, f, g, b_min, b_max, device=dev)
            for e in range(E):
                gen.manual_seed(50_000_017 * (l + 1) + 2 * e)
                api.pack_mwq(torch.randn((1, 2 * f, d), generator=gen, device=dev) * 0.02,
                             w13.expert(e))
                gen.manual_seed(50_000_017 * (l + 1) + 2 * e + 1)
                api.pack_mwq(torch.randn((1, d, f), generator=gen, device=dev) * 0.02,
                             w2.expert(e))
            gen.manual_seed(5000 + l)
            Wg = torch.randn((E, d), generator=gen, device=dev) * 0.02
            stack.append((w13, w2, Wg, api.Routing.empty(T, E, k, b_min, b_max, device=dev)))
        torch.cuda.synchronize()
        rng = np.random.default_rng(5)
        tiers = rng.choice(np.array([2, 4, 8], np.uint8), size=(T, 1))
        table = torch.from_numpy(np.repeat(tiers, E, axis=1)).to(dev)
        req = torch.arange(T, dtype=torch.int32, device=dev)
        x0 = torch.from_numpy(rng.standard_normal((T, d), dtype=np.float32)).to(dev)
        x = x0.clone()
        h = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, d, f, E, k), dtype=torch.uint8, device=dev)

        def decode_step():
            for w13, w2, Wg, r in stack:
                api.route(h, Wg, None, k, req, table, b_min, b_max, out=r)
                api.moe_forward(h, w13, w2, r, k, out=y, workspace=ws)
                api.residual_rmsnorm(x, y, eps, h=h)

        api.residual_rmsnorm(x, None, eps, h=h)
        warm(lambda i: decode_step(), 1)   # warm-up steps, then restart from x0
        x.copy_(x0)
        api.residual_rmsnorm(x, None, eps, h=h)
        torch.cuda.synchronize()
        t_start = torch.cuda.Event(enable_timing=True)
        t_stop = torch.cuda.Event(enable_timing=True)
        t_start.record()
        for _ in range(steps):
            decode_step()
        t_stop.record()
        torch.cuda.synchronize()
        ms = t_start.elapsed_time(t_stop)
        step_bytes = 0
        for w13, w2, Wg, r in stack:
            for b in r.expert_maxbit.cpu().numpy():
                step_bytes += mwq_bytes(2 * f, d, g, b_min, int(b)) + mwq_bytes(d, f, g, b_min, int(b))
        gbps = step_bytes * steps / (ms * 1e-3) / 1e9
        finite = bool(torch.isfinite(x).all().item())
        del stack
        torch.cuda.empty_cache()
        return {"workload": f"{n_layers}-layer decoder stack of Mixtral-8x7B-shaped MoE layers "
                            f"(x <- x + MoE(rmsnorm(x)), attention absent), {T} sequences x "
                            f"{steps} decode steps, per-sequence bit tier from {{2,4,8}}, "
                            f"group 128, 8-bit nest, all layers resident",
                "layers": n_layers, "sequences": T, "steps": steps,
                "ms_total": round(ms, 2), "ms_per_step": round(ms / steps, 4),
                "tokens_per_s": round(T * steps / (ms * 1e-3), 1),
                "alg_bytes_per_step": step_bytes, "hbm_GBps": round(gbps, 1),
                "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "hidden_state_finite": finite}

    def run_variant(label, dV, fV, EV, kV, bmin, bmax, choices, probs, copies, steps, warmup=5,
                    T=16):
        """Batch-T decode of a layer of another shape or nest: `copies`
        rotating packed copies, per-(request, expert) bit tables drawn from
        `choices` with `probs`.  Reports the step and the W1/W3 kernel's HBM
        rate (HIP events on the launch stream) against its algorithmic bytes."""
        sets = []
        for c in range(copies):
            w13 = api.MWQ.empty(EV, 2 * fV, dV, g, bmin, bmax, device=dev)
            w2 = api.MWQ.empty(EV, dV, fV, g, bmin, bmax, device=dev)
            for e in range(EV):
                gen.manual_seed(90_000_049 * (c + 1) + 2 * e)
                api.pack_mwq(torch.randn((1, 2 * fV, dV), generator=gen, device=dev) * 0.02,
                             w13.expert(e))
                gen.manual_seed(90_000_049 * (c + 1) + 2 * e + 1)
                api.pack_mwq(torch.randn((1, dV, fV), generator=gen, device=dev) * 0.02,
                             w2.expert(e))
            gen.manual_seed(9000 + c)
            Wg = torch.randn((EV, dV), generator=gen, device=dev) * 0.02
            sets.append((w13, w2, Wg, api.Routing.empty(T, EV, kV, bmin, bmax, device=dev)))
        rng = np.random.default_rng(11 + T + bmin)
        x = torch.from_numpy(rng.standard_normal((T, dV), dtype=np.float32)).to(dev).to(torch.bfloat16)
        req = torch.arange(T, dtype=torch.int32, device=dev)
        tables = [torch.from_numpy(rng.choice(np.array(choices, np.uint8), size=(T, EV),
                                              p=probs)).to(dev) for _ in range(copies)]
        out = torch.empty((T, dV), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, dV, fV, EV, kV), dtype=torch.uint8,
                         device=dev)

        def step(i, events=None):
            w13, w2, Wg, r = sets[i % copies]
            api.route(x, Wg, None, kV, req, tables[i % copies], bmin, bmax, out=r)
            api.moe_forward(x, w13, w2, r, kV, out=out, workspace=ws, events=events)

        w0 = warm(step, warmup)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
        for row in evs:
            for ev in row:
                ev.record()
        torch.cuda.synchronize()
        t_start = torch.cuda.Event(enable_timing=True)
        t_stop = torch.cuda.Event(enable_timing=True)
        t_start.record()
        for i in range(steps):
            step(w0 + i, evs[i])
        t_stop.record()
        torch.cuda.synchronize()
        ms = t_start.elapsed_time(t_stop) / steps
        alg13 = [sum(mwq_bytes(2 * fV, dV, g, bmin, int(b))
                     for b in sets[c][3].expert_maxbit.cpu().numpy()) for c in range(copies)]
        b13 = float(np.mean([alg13[(w0 + i) % copies] for i in range(steps)]))
        d13 = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
        gbps = b13 / (d13 * 1e-3) / 1e9
        del sets
        torch.cuda.empty_cache()
        return {"workload": label, "tokens": T, "ms_per_step": round(ms, 4),
                "tokens_per_s": round(T / (ms * 1e-3), 1), "w13_ms": round(d13, 4),
                "w13_alg_bytes": b13, "w13_GBps": round(gbps, 1),
                "w13_hbm_frac": round(gbps / HBM_PEAK_GBPS, 4)}

    def run_learned(T, steps, warmup=5):
        """The batch-T decode step of the rotating layers with the learned
        bit-width routers of Sec. 3.2 in place of the width table (one linear
        router per expert over the 7 widths of the nest, seeded Gaussian
        weights), and the routing calls alone with either source of widths.
        Reports the step time and the routers' share of it."""
        L_ = b_max - b_min + 1
        rng = np.random.default_rng(17 + T)
        x = torch.from_numpy(rng.standard_normal((T, d), dtype=np.float32)).to(dev).to(torch.bfloat16)
        req = torch.arange(T, dtype=torch.int32, device=dev)
        table = torch.from_numpy(rng.choice(np.array([2, 3, 4, 8], np.uint8), size=(T, E),
                                            p=[0.2, 0.3, 0.3, 0.2])).to(dev)
        routers = []
        for l in range(NL):
            gen.manual_seed(3_000_000 + l)
            routers.append((torch.randn((E, L_, d), generator=gen, device=dev) * 0.05,
                            torch.randn((E, L_), generator=gen, device=dev) * 0.05))
        r = api.Routing.empty(T, E, k, b_min, b_max, device=dev)
        bl = torch.empty((T, E, L_), dtype=torch.float32, device=dev)
        out = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, d, f, E, k), dtype=torch.uint8, device=dev)

        def route_l(i):
            w13, w2, Wg = layers[i % NL]
            api.route_learned(x, Wg, None, k, routers[i % NL][0], routers[i % NL][1], b_min,
                              b_max, out=r, bit_logits=bl)

        def route_t(i):
            api.route(x, layers[i % NL][2], None, k, req, table, b_min, b_max, out=r)

        def step(i):
            route_l(i)
            w13, w2, Wg = layers[i % NL]
            api.moe_forward(x, w13, w2, r, k, out=out, workspace=ws)

        def timed(fn, n):
            w0 = warm(fn, warmup)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for i in range(n):
                fn(w0 + i)
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / n

        ms = timed(step, steps)
        ms_rl = timed(route_l, steps)
        ms_rt = timed(route_t, steps)
        bits = r.topk_bits.cpu().numpy().ravel()
        return {"workload": f"Mixtral-8x7B-shaped MoE layer decode, batch {T}, bit-widths from "
                            f"learned per-expert routers over the 2..8 nest (seeded weights), "
                            f"{NL} rotating layers",
                "tokens": T, "ms_per_step": round(ms, 4), "tokens_per_s": round(T / (ms * 1e-3), 1),
                "route_ms_learned": round(ms_rl, 4), "route_ms_table": round(ms_rt, 4),
                "router_share_of_step": round((ms_rl - ms_rt) / ms, 4),
                "widths_used_last_step": np.bincount(bits, minlength=b_max + 1)[b_min:].tolist()}

    def run_tiny(steps, warmup=10):
        """The tiny layer: d_model 256, d_ff 512, 8 SwiGLU experts top-2,
        64 tokens of fp32 activations N(0,1), weights N(0, 0.02) packed with
        group 64 nested to 8 bits, one request with bits per expert uniform
        from {2,4,8} (seed 0).  All of its weights fit in the caches, so it
        carries no roofline claim: route + forward time only."""
        dT, fT, ET, kT, gT, T = 256, 512, 8, 2, 64, 64
        rng = np.random.default_rng(0)
        x = torch.from_numpy(rng.standard_normal((T, dT), dtype=np.float32)).to(dev)
        w13 = api.MWQ.empty(ET, 2 * fT, dT, gT, b_min, b_max, device=dev)
        w2 = api.MWQ.empty(ET, dT, fT, gT, b_min, b_max, device=dev)
        gen.manual_seed(0)
        api.pack_mwq(torch.randn((ET, 2 * fT, dT), generator=gen, device=dev) * 0.02, w13)
        api.pack_mwq(torch.randn((ET, dT, fT), generator=gen, device=dev) * 0.02, w2)
        Wg = torch.randn((ET, dT), generator=gen, device=dev) * 0.02
        table = torch.from_numpy(rng.choice(np.array([2, 4, 8], np.uint8), size=(1, ET))).to(dev)
        r = api.Routing.empty(T, ET, kT, b_min, b_max, device=dev)
        out = torch.empty((T, dT), dtype=torch.float32, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, dT, fT, ET, kT), dtype=torch.uint8,
                         device=dev)

        def step(i):
            api.route(x, Wg, None, kT, None, table, b_min, b_max, out=r)
            api.moe_forward(x, w13, w2, r, kT, out=out, workspace=ws)

        w0 = warm(step, warmup)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(steps):
            step(w0 + i)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        return {"workload": "tiny MoE layer (d_model 256, d_ff 512, 8 SwiGLU experts top-2, 64 "
                            "tokens of fp32 activations, group 64, 8-bit nest, bits per expert "
                            "from {2,4,8}); computed on bf16/fp8-piece operands with fp32 "
                            "accumulation; cache-resident, no roofline claim",
                "tokens": T, "ms_per_step": round(ms, 4), "tokens_per_s": round(T / (ms * 1e-3), 1)}

    def run_ceiling(gib, reps=10):
        """This GPU's HBM read ceiling: a plain kernel that streams `gib` GiB
        once with 16-byte nontemporal loads (d2moe_stream_read), timed with
        HIP events; best and median of `reps` reads."""
        n = int(gib * (1 << 30)) // 16 * 16
        buf = torch.empty(n // 4, dtype=torch.int32, device=dev)
        buf.fill_(1)
        best = None
        for blocks in (1024, 2048, 4096, 8192, 32768):
            sink = torch.empty(blocks, dtype=torch.int32, device=dev)
            warm(lambda i: api.stream_read(buf, sink), 1, min_ms=20.0)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
            ev[0].record()
            for i in range(reps):
                api.stream_read(buf, sink)
                ev[i + 1].record()
            torch.cuda.synchronize()
            rates = np.array([n / (ev[i].elapsed_time(ev[i + 1]) * 1e-3) / 1e9
                              for i in range(reps)])
            if best is None or np.median(rates) > np.median(best[1]):
                best = (blocks, rates)
        del buf
        torch.cuda.empty_cache()
        blocks, rates = best
        return {"kernel": f"plain streaming read of {gib:g} GiB, 16-byte nontemporal loads, "
                          f"{blocks} workgroups of 256 threads (best of 1024-32768)",
                "best_GBps": round(float(rates.max()), 1),
                "median_GBps": round(float(np.median(rates)), 1),
                "median_frac_of_peak": round(float(np.median(rates)) / HBM_PEAK_GBPS, 4)}

    def run_calib(tokens=2048, corr=0.8, gamma=128):
        """Calibration-aware MWQ setup at the Mixtral shapes: the binary64 factor
        of the regularised Hessian of `tokens` synthetic calibration tokens
        (AR(1) feature correlation `corr`, lambda 1 % of the mean Hessian
        diagonal) for the W1/W3 input (4096 features) and the W2 input (14336),
        and the calibrated pack of one expert of each (blocks of 128 columns,
        nest 2..8).  Setup work, untimed in the layer step; reported with the
        binary32 rate of the compensation arithmetic (2 flops per fmaf of
        E U_BF, summed over levels and blocks) against the chip's fp32 vector
        peak."""
        res = {}
        for name, h, N in (("w13", d, 2 * f), ("w2", f, d)):
            rng = np.random.default_rng(31 + h)
            Z = rng.standard_normal((tokens, h), dtype=np.float32)
            X = np.empty_like(Z)
            X[:, 0] = Z[:, 0]
            c2 = np.float32(np.sqrt(1 - corr * corr))
            for c in range(1, h):
                X[:, c] = np.float32(corr) * X[:, c - 1] + c2 * Z[:, c]
            lam = 0.01 * float(np.mean(2.0 * np.sum(X.astype(np.float64) ** 2, axis=0)))
            Xd = torch.from_numpy(X).to(dev)
            gen.manual_seed(77_000 + h)
            W = torch.randn((1, N, h), generator=gen, device=dev) * 0.02
            m = api.MWQ.empty(1, N, h, g, b_min, b_max, device=dev)
            api.mwq_calib_factor(Xd[:128], lam)          # first launches, untimed
            torch.cuda.synchronize()
            a, b, c_ = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            a.record()
            U, info = api.mwq_calib_factor(Xd, lam)
            b.record()
            api.pack_mwq_calibrated(W, U, gamma, m)
            c_.record()
            torch.cuda.synchronize()
            ms_f, ms_p = a.elapsed_time(b), b.elapsed_time(c_)
            levels = b_max - b_min + 1
            flop = 2.0 * N * levels * sum(gamma * (h - b0 - gamma) for b0 in range(0, h, gamma))
            res[name] = {"rows": N, "cols": h, "factor_ms": round(ms_f, 2),
                         "factor_ok": int(info.item()) == 0,
                         "calibrated_pack_ms": round(ms_p, 2),
                         "compensation_TFLOPs": round(flop / (ms_p * 1e-3) / 1e12, 2),
                         "fp32_vector_peak_TFLOPs": 157.3,
                         "frac": round(flop / (ms_p * 1e-3) / 1e12 / 157.3, 4)}
            del W, U, Xd, m
            torch.cuda.empty_cache()
        res["workload"] = (f"calibration-aware MWQ setup, one Mixtral-8x7B-shaped expert's W1/W3 "
                           f"(28672 x 4096) and W2 (4096 x 14336), {tokens} synthetic calibration "
                           f"tokens (AR(1) correlation {corr}), blocks of {gamma} columns, group "
                           f"128, nest 2..8")
        return res

    def run_streamed(steps, T=16):
        """One Mixtral-8x7B-shaped layer (8-bit nest, group 128) whose packed
        experts live in pinned host memory and are streamed into a device copy
        for each step (the device copy starts empty every step, as when the
        layer does not stay resident), batch T, bits from {2,3,4,8}: the
        units of the step in HEBF order and in ascending expert order
        (Sec. 3.4.3, Fig. 9), each unit's nested delta copied on an I/O
        stream and its bucket computed when it lands.  Reported with the
        bytes copied and the rate of a plain pinned host-to-device copy of
        the same size measured in the same run."""
        w13, w2, Wg = layers[0]

        def pin(t):
            h_ = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
            h_.copy_(t)
            return h_

        def host_copy(m):
            return api.MWQ(m.n_experts, m.rows, m.cols, m.group, m.b_min, m.b_max,
                           pin(m.planes), pin(m.scales), pin(m.zeros))

        h13, h2 = host_copy(w13), host_copy(w2)
        d13 = api.MWQ.empty(E, 2 * f, d, g, b_min, b_max, device=dev)
        d2 = api.MWQ.empty(E, d, f, g, b_min, b_max, device=dev)
        rng = np.random.default_rng(41)
        x = torch.from_numpy(rng.standard_normal((T, d), dtype=np.float32)).to(dev).to(torch.bfloat16)
        req = torch.arange(T, dtype=torch.int32, device=dev)
        table = torch.from_numpy(rng.choice(np.array([2, 3, 4, 8], np.uint8), size=(T, E),
                                            p=[0.2, 0.3, 0.3, 0.2])).to(dev)
        r = api.route(x, Wg, None, k, req, table, b_min, b_max)
        hist = r.hist.cpu().numpy()
        io = torch.cuda.Stream()
        out = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(api.moe_forward_workspace(T, d, f, E, k), dtype=torch.uint8, device=dev)

        def ascending():
            units, Lv = [], b_max - b_min + 1
            for j in range(E):
                have = 0
                for kk in range(Lv):
                    if hist[j, kk] > 0:
                        b = b_min + kk
                        units.append((j, b, have, max(have, b), int(hist[j, kk])))
                        have = max(have, b)
            return units

        orders = {"hebf": api.hebf_order(hist, b_min, b_max), "ascending": ascending()}
        evs = [torch.cuda.Event() for _ in range(E * (b_max - b_min + 1))]
        res = {}
        for name, units in orders.items():
            times = []
            for i in range(steps + 1):
                resident = np.zeros(E, np.uint8)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                api.moe_forward_streamed(x, h13, h2, d13, d2, resident, r, k, hist, units,
                                         evs[:len(units)], io, out=out, workspace=ws)
                torch.cuda.synchronize()
                if i > 0:
                    times.append((time.perf_counter() - t0) * 1e3)
            res[name] = round(float(np.median(times)), 3)
        nbytes = sum(mwq_bytes(2 * f, d, g, b_min, int(b)) + mwq_bytes(d, f, g, b_min, int(b))
                     for b in r.expert_maxbit.cpu().numpy())
        src = torch.empty(nbytes // 4, dtype=torch.int32, pin_memory=True)
        dst = torch.empty(nbytes // 4, dtype=torch.int32, device=dev)
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        ct = []
        for _ in range(3):
            t0 = time.perf_counter()
            dst.copy_(src, non_blocking=True)
            torch.cuda.synchronize()
            ct.append((time.perf_counter() - t0) * 1e3)
        copy_ms = float(np.median(ct))
        del h13, h2, d13, d2, src, dst
        torch.cuda.empty_cache()
        return {"workload": f"Mixtral-8x7B-shaped MoE layer decode, batch {T}, bits from "
                            f"{{2,3,4,8}}, experts streamed from pinned host memory into an empty "
                            f"device copy each step (nested delta planes per unit)",
                "tokens": T, "units": len(orders["hebf"]), "bytes_streamed": int(nbytes),
                "ms_per_step_hebf": res["hebf"], "ms_per_step_ascending": res["ascending"],
                "plain_h2d_copy_ms": round(copy_ms, 3),
                "h2d_GBps_plain": round(nbytes / (copy_ms * 1e-3) / 1e9, 1),
                "h2d_GBps_streamed_hebf": round(nbytes / (res["hebf"] * 1e-3) / 1e9, 1)}

    main_res = run_batch(args.batch, args.steps, args.warmup, profile=True)
    if args.dump_steps:
        print("per-step ms:", main_res["per_step_ms"], file=sys.stderr)
        print("per-step W1/W3 ms:", main_res["per_step_w13_ms"], file=sys.stderr)
    for key in ("per_step_ms", "per_step_w13_ms"):
        main_res.pop(key, None)
    learned = run_learned(args.batch, max(args.steps // 2, 10)) if args.learned else None
    sweep = []
    for T in [int(v) for v in args.sweep.split(",") if v.strip()]:
        r = run_batch(T, max(args.steps // 2, 5), args.warmup, profile=True)
        sweep.append({kk: (round(v, 4) if isinstance(v, float) else v) for kk, v in r.items()})

    ceiling = run_ceiling(args.ceiling_gib) if args.ceiling_gib > 0 else None
    calib = run_calib() if args.calib else None
    streamed = run_streamed(args.stream_steps) if args.stream_steps > 0 else None
    tiny = run_tiny(args.tiny_steps) if args.tiny_steps > 0 else None
    prefill = run_prefill(args.prefill_steps, 2) if args.prefill_steps > 0 else None
    fine = run_fine(args.fine_steps, 2) if args.fine_steps > 0 else None
    stack_res = run_stack(args.stack_steps) if args.stack_steps > 0 else None
    variants = None
    if args.variant_steps > 0:
        vs = args.variant_steps
        variants = {
            "v1": run_variant("Mixtral-8x7B-shaped MoE layer decode, batch 16, the paper's first "
                              "nest (b 2-4, bits {2,3,4} p {.3,.4,.3}), group 128, 4 rotating "
                              "copies", d, f, E, k, 2, 4, (2, 3, 4), (0.3, 0.4, 0.3), 4, vs),
            "v2": run_variant("Mixtral-8x7B-shaped MoE layer decode, batch 16, the paper's "
                              "second nest (b 5-8, bits {5,6,7,8} p .25 each), group 128, 4 "
                              "rotating copies", d, f, E, k, 5, 8, (5, 6, 7, 8),
                              (0.25, 0.25, 0.25, 0.25), 4, vs),
            "dense": run_variant("LLaMA2-13B-shaped dense SwiGLU FFN (d_model 5120, d_ff 13824; "
                                 "one expert, top-1) decode, batch 16, per-request bits {2,3,4} "
                                 "p {.3,.4,.3} of the first nest, group 128, 8 rotating copies",
                                 5120, 13824, 1, 1, 2, 4, (2, 3, 4), (0.3, 0.4, 0.3), 8, vs),
        }

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(d, f, E, k, g)

    traffic = profiled_traffic()
    line = {
        "metric": METRIC,
        "value": round(main_res["tokens_per_s"], 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_res["ms_per_step"], 5),
        "ms_per_step_eager": round(main_res["ms_per_step_eager"], 5),
        "launch": "hip graph per layer step" if use_graphs else "eager",
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"Mixtral-8x7B-shaped MoE layer decode (d_model 4096, d_ff 14336, "
                               f"8 SwiGLU experts, top-2), batch {args.batch}, MWQ group 128 nested "
                               f"to 8 bits, per-(request,expert) bits from {{2,3,4,8}} p "
                               f"{{.2,.3,.3,.2}}, {NL} rotating layers",
                   "batch": args.batch, "d_model": d, "d_ff": f, "experts": E, "top_k": k,
                   "group": g},
        "warmup_steps_run": main_res["warmup_steps_run"],
        "step_ms_p10_p50_p90": main_res["step_ms_p10_p50_p90"],
        "hbm_GBps": round(main_res["layer_GBps"], 1),
        "hbm_frac": round(main_res["layer_GBps"] / HBM_PEAK_GBPS, 4),
        "roofline": {"bound": "hbm", "kernel": "W1/W3 expert kernel",
                     "achieved": round(main_res["w13_GBps"], 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(main_res["w13_GBps"] / HBM_PEAK_GBPS, 4),
                     "traffic": traffic[0],
                     "traffic_unit": "bytes/launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "alg_bytes_per_launch": main_res["w13_bytes"],
                     "avg_ms": round(main_res["w13_ms"], 5),
                     "ms_p10_p50_p90": main_res["w13_ms_p10_p50_p90"],
                     "stream_read_ceiling": ceiling},
        "w2_kernel": {"achieved": round(main_res["w2_GBps"], 1), "avg_ms": round(main_res["w2_ms"], 5),
                      "traffic": traffic[1]},
        "sweep": sweep,
        "tiny": tiny,
        "prefill": prefill,
        "fine_grained": fine,
        "stack": stack_res,
        "variants": variants,
        "learned_router": learned,
        "calibrated_mwq": calib,
        "streamed": streamed,
        "cpu_baseline": cpu,
        "pack_seconds": round(pack_s, 2),
    }
    print(json.dumps(line), flush=True)


PROFILE = os.path.join(ROOT, "profiles", "decode_step_mixtral_T16_hbm_bytes.txt")


def kernel_source_hash() -> str:
    """Hash of the decode kernels' code (ffn_decode.hip and internal.h with
    comments and blank space removed, so that editing a comment does not
    mark the committed byte counters as stale)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in ("ffn_decode.hip", "internal.h"):
        with open(os.path.join(ROOT, "paper_2504_15299_amd", "csrc", name)) as fh:
            code = fh.read()
        code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
        code = re.sub(r"//[^\n]*", " ", code)
        h.update(" ".join(code.split()).encode())
    return h.hexdigest()[:16]


def profiled_traffic():
    """HBM bytes per launch of the W1/W3 and W2 decode kernels from the
    committed rocprofv3 counter summary, or None when the kernel source has
    changed since the counters were taken (or no summary exists)."""
    try:
        with open(PROFILE) as fh:
            kv = dict(line.split(": ", 1) for line in fh.read().splitlines() if ": " in line)
    except OSError:
        return None, None
    if kv.get("kernel_source_sha256_16", "").strip() != kernel_source_hash():
        return None, None
    return int(kv["traffic_w13_bytes"]), int(kv["traffic_w2_bytes"])


def host_cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(d, f, E, k, g, n_tokens=4):
    """The CPU oracle (single thread, as it stands) on a bounded sample of the
    decode workload: n_tokens decode tokens of the same layer shape, one
    request each with bits per expert from {2,3,4,8}; gate logits and dual
    routing (timed as `route`), each token's selected experts' SwiGLU FFNs
    from their MWQ codes and the combine (timed as `forward`).  Quantizing
    the experts is setup and is not timed.  The process is pinned to one
    host CPU for the timed part (and unpinned afterwards)."""
    import numpy as np

    from oracle import oracle as O

    rng = np.random.default_rng(11)
    x = rng.standard_normal((n_tokens, d), dtype=np.float32)
    Wg = (rng.standard_normal((E, d), dtype=np.float32) * 0.02)
    table = rng.choice(np.array([2, 3, 4, 8], np.uint8), size=(n_tokens, E),
                       p=[0.2, 0.3, 0.3, 0.2]).astype(np.uint8)
    req = np.arange(n_tokens, dtype=np.int32)
    route = O.route_from_logits(O.gate_logits(x, Wg), k, req, table)
    codes13, codes2 = {}, {}
    for e in sorted({int(e) for e in route["topk_idx"].ravel()}):
        codes13[e] = O.mwq_quantize((rng.standard_normal((2 * f, d), dtype=np.float32) * 0.02), g)
        codes2[e] = O.mwq_quantize((rng.standard_normal((d, f), dtype=np.float32) * 0.02), g)
    allowed = sorted(os.sched_getaffinity(0))
    cpu = allowed[0]
    os.sched_setaffinity(0, {cpu})
    try:
        t0 = time.perf_counter()
        route = O.route_from_logits(O.gate_logits(x, Wg), k, req, table)
        t1 = time.perf_counter()
        for t in range(n_tokens):
            ys = []
            for i in range(k):
                e = int(route["topk_idx"][t, i])
                ys.append(O.expert_ffn(codes13[e], codes2[e], int(route["topk_bits"][t, i]),
                                       x[t:t + 1].astype(np.float64))[0])
            O.combine(route["topk_w"][t:t + 1], np.stack(ys)[None])
        t2 = time.perf_counter()
    finally:
        os.sched_setaffinity(0, set(allowed))
    secs = t2 - t0
    ncpu = os.cpu_count()
    return {"value": round(n_tokens / secs, 5), "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "seconds": round(secs, 3), "route_seconds": round(t1 - t0, 4),
            "forward_seconds": round(t2 - t1, 3),
            "host": f"oracle on 1 of {ncpu} host cores (pinned to CPU {cpu}; "
                    f"{len(allowed)} in this process's affinity), {host_cpu_model()}",
            "host_cores": ncpu, "cpu_model": host_cpu_model(),
            "sample": f"{n_tokens} decode tokens of the same layer shape, one request each "
                      f"(gate, routing, each token's 2 experts' SwiGLU FFNs from MWQ codes at "
                      f"bits from {{2,3,4,8}}, combine); expert quantization untimed"}


if __name__ == "__main__":
    main()
