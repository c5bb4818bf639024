"""Benchmark: garbled scaling gadgets evaluated per second on one MI355X.

A step is one call of redash_eval_scale over the whole workload (the online
phase of the gadget; garbling and encoding happen before the timed region,
decoding after it).  Default workload: the batched conv map, 16x64x56x56 =
3,211,264 gadgets over the first 12 primes, scaled by 37.

Prints one JSON line on stdout; progress goes to stderr.
"""

from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "garbled scaling gadgets evaluated/sec (1 GPU) + % HBM roofline"
HBM_PEAK_GBS = 8000.0
# int32 vector ALU: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (one lane-op per lane per clock)
ALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# LDS: 128 bytes per clock per CU (32 banks x 4 bytes)
LDS_PEAK_GBS = 256 * 128 * 2.4e9 / 1e9


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def oracle_rate(w, x, sample: int, target_s: float):
    """The CPU oracle's evaluation, single-threaded, on the first `sample`
    gadgets of workload w (garbled by the oracle, untimed), repeated until
    about target_s seconds have been timed; checked by decode afterwards.
    Returns (gadgets/s, passes, seconds timed)."""
    from oracle import oracle as O

    op = O.make_params(list(w.moduli), list(w.scale_idx), sample, w.seed)
    t0 = time.time()
    offs, zin, zout, tab = O.garble(op, 0, sample)
    X = O.encode(op, x[:sample], zin, offs)
    log(f"cpu baseline: oracle garbled {sample} gadgets of {w.name} in {time.time() - t0:.1f} s")
    reps, elapsed = 0, 0.0
    while elapsed < target_s:
        t1 = time.perf_counter()
        Y = O.evaluate(op, 0, sample, X, tab)
        elapsed += time.perf_counter() - t1
        reps += 1
    y, bad = O.decode(op, Y, zout, offs)
    assert bad.sum() == 0 and np.array_equal(y, expected_values(w, x[:sample]))
    return sample * reps / elapsed, reps, elapsed


def cpu_baseline(w, x, sample: int, target_s: float, slices: bool = True):
    """The oracle's evaluation rate on the benchmark workload (a slice of its
    first gadgets; gadgets are independent, so the rate carries over), and on
    slices of the other workloads: the tiny and dense ones whole, the first
    gadgets of the conv map and of three ResNet-18 layers (the stem, a layer-4
    conv scaled by 31 x 37, the fc layer)."""
    rate, reps, elapsed = oracle_rate(w, x, sample, target_s)
    out = {
        "value": round(rate, 1),
        "unit": "gadgets/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"oracle eval of the first {sample} gadgets of the {w.name} workload "
                  f"(oracle-garbled tables), {reps} passes, {elapsed:.1f} s timed; plain C, one thread; "
                  f"host has {len(os.sched_getaffinity(0))} cores available",
    }
    if slices:
        from paper_2506_14489_amd import workloads as WL

        plan = [(WL.TINY, 1024), (WL.DENSE, 4096), (WL.CONV, 2048),
                (WL.by_name("resnet18.stem"), 1024), (WL.by_name("resnet18.l4.1.b"), 1024),
                (WL.by_name("resnet18.fc"), 1000)]
        out["slices"] = []
        for sw, count in plan:
            sx = WL.make_inputs(sw)
            r, k, t = oracle_rate(sw, sx, count, max(target_s / 6, 1.0))
            out["slices"].append({"workload": sw.name, "gadgets": count, "of": sw.n, "value": round(r, 1),
                                  "unit": "gadgets/s", "passes": k, "seconds": round(t, 2)})
    return out


def expected_values(w, x):
    """What the gadget returns: floor((x + r)/s) with r = floor(P/2) mod s
    (the shift constants floor(P/2) and floor(floor(P/2)/s) of Sec. 3.4;
    r = 0, i.e. floor(x/s), whenever P/(2s) is an integer)."""
    return np.floor_divide(x + (w.P // 2) % w.s, w.s)


MFMA_I8_PEAK_TOPS = 5000.0  # dense int8 matrix-core peak of the MI355X, TOP/s


_VALUES = {}


def layer_values(w):
    """WL.make_inputs(w), computed once per workload (the exact conv outputs of
    a ResNet-18 layer serve both its linear layer's check and its gadget)."""
    from paper_2506_14489_amd import workloads as WL

    if w not in _VALUES:
        _VALUES[w] = WL.make_inputs(w)
    return _VALUES[w]


def time_linear_layer(w, params, buf, steps: int, warmup: int, dev, garble: bool = True):
    """The garbled conv layer that produces workload w's activations (Y = sum w X
    on the labels of its int8 inputs), on the gadget's garbled input labels:
    prepare the weights, garble the output zero-labels, time the evaluator,
    decode every output.  Returns a summary dict."""
    import torch

    from paper_2506_14489_amd import binding as B
    from paper_2506_14489_amd import cost
    from paper_2506_14489_amd import workloads as WL

    a, wt = WL.layer_operands(w)
    if w.kind == "fc":  # a dense layer: 1x1 kernel over `batch` positions of one row
        (n, c_in), (c_out, _) = w.in_shape, w.w_shape
        h, wd, kh, kw, stride, pad = 1, 1, 1, 1, 1, 0
        lp = B.make_linear_params(w.moduli, n, c_in, 1, 1, c_out)
    else:
        n, c_in, h, wd = w.in_shape
        c_out, _, kh, kw = w.w_shape
        stride, pad = w.stride, w.pad
        lp = B.make_linear_params(w.moduli, n, c_in, h, wd, c_out, kh, kw, stride, pad)
    sz = B.redash_linear_plan(lp)
    stream = torch.cuda.current_stream()
    n_in = n * c_in * h * wd
    assert n_in == params.n, "the layer's inputs reuse the gadget's garbled labels"
    X = torch.empty_like(buf.in_labels)
    B.redash_encode(params, torch.from_numpy(a.reshape(-1).astype(np.int64)).to(dev), buf.in_zero, buf.offsets, X,
                    stream)
    prep = torch.empty(sz["prepared_bytes"], dtype=torch.uint8, device=dev)
    work = torch.empty(sz["work_bytes"], dtype=torch.uint8, device=dev)
    B.redash_linear_prepare(lp, torch.from_numpy(wt.astype(np.int32)).to(dev), prep, stream)
    Y = torch.empty(sz["out_label_words"], dtype=torch.int32, device=dev)
    Z = torch.empty_like(Y)
    B.redash_linear_garble(lp, buf.in_zero, prep, None, buf.offsets, work, Z, stream)
    gc.collect()
    t_w, done = time.perf_counter(), 0  # as time_workload: at least `warmup` calls and 50 ms
    while done < warmup or time.perf_counter() - t_w < 0.05:
        B.redash_linear_eval(lp, X, prep, work, Y, stream)
        done += 1
        if done % 8 == 0:
            torch.cuda.synchronize()
    # An event recorded behind a still-running kernel is stamped when that kernel
    # starts (measured: 10 calls timed that way take 11 calls' time), so the
    # warm-up calls are waited for before the first event.
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        B.redash_linear_eval(lp, X, prep, work, Y, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    g0 = torch.cuda.Event(enable_timing=True)
    g1 = torch.cuda.Event(enable_timing=True)
    if garble:
        g0.record(stream)
        B.redash_linear_garble(lp, buf.in_zero, prep, None, buf.offsets, work, Z, stream)
        g1.record(stream)
    n_out = w.n
    dp = B.make_params(w.moduli, w.scale_idx, n_out, w.seed)
    y = torch.empty(n_out, dtype=torch.int64, device=dev)
    bad = torch.zeros(1, dtype=torch.int64, device=dev)
    B.redash_decode(dp, Y, Z, buf.offsets, y, bad, stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    ok = int(bad.item()) == 0 and np.array_equal(y.cpu().numpy(), layer_values(w))
    if not ok:
        log(f"linear layer {w.name}: decode check FAILED")
        sys.exit(1)
    ops = cost.linear_ops_per_output(w.moduli, c_in, kh, kw) * n_out
    tops = ops / (ms / 1e3) / 1e12
    gbs = cost.linear_bytes(w.moduli, n_in, n_out) / (ms / 1e3) / 1e9
    log(f"linear layer {w.name}: eval {ms:.3f} ms per call, {tops:.0f} TOP/s")
    r = {
        "layer": (f"dense {c_in}->{c_out}, batch {n}" if w.kind == "fc" else
                  f"conv {kh}x{kw} stride {stride} pad {pad}, {c_in}->{c_out} channels, input {list(w.in_shape)}")
                 + f", {len(w.moduli)} moduli",
        "ms_per_call": round(ms, 4),
        "outputs_per_s": round(n_out / (ms / 1e3), 1),
        "roofline": {"bound": "mfma", "achieved": round(tops, 1), "peak": MFMA_I8_PEAK_TOPS, "unit": "TOP/s",
                     "frac": round(tops / MFMA_I8_PEAK_TOPS, 4), "dtype": "i8",
                     "ops_per_output": cost.linear_ops_per_output(w.moduli, c_in, kh, kw), "kernel": "k_linear"},
        "hbm": {"achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4)},
        "check": "decode(eval labels, garbler zero-labels) = exact integer convolution, all outputs",
        "steps": steps,
    }
    if garble:
        r["garble_ms"] = round(g0.elapsed_time(g1), 4)
    return r


def time_resnet18_linear(steps: int, warmup: int, dev):
    """The 21 garbled linear layers of ResNet-18 at batch 1 (20 convolutions and
    the dense layer), each on input labels garbled for its own input size:
    sum of the per-layer evaluation times, every output decoded and checked."""
    import torch

    from paper_2506_14489_amd import binding as B
    from paper_2506_14489_amd import cost
    from paper_2506_14489_amd import workloads as WL

    layers, ms_tot, ops_tot = [], 0.0, 0
    for w in WL.RESNET18:
        n_in = int(np.prod(w.in_shape))
        params = B.make_params(w.moduli, w.scale_idx, n_in, w.seed)
        buf = B.Buffers(params, dev)
        B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work,
                              torch.cuda.current_stream())
        r = time_linear_layer(w, params, buf, steps, warmup, dev, garble=False)
        c_in = w.in_shape[1]
        kh, kw = (1, 1) if w.kind == "fc" else w.w_shape[2:]
        ops_tot += cost.linear_ops_per_output(w.moduli, c_in, kh, kw) * w.n
        ms_tot += r["ms_per_call"]
        layers.append({"layer": w.name, "shape": r["layer"], "ms_per_call": r["ms_per_call"],
                       "int8_frac": r["roofline"]["frac"]})
        del buf
        torch.cuda.empty_cache()
    tops = ops_tot / (ms_tot / 1e3) / 1e12
    log(f"resnet18 linear layers: {ms_tot:.3f} ms over {len(layers)} layers")
    return {
        "ms_total": round(ms_tot, 4),
        "int8_frac": round(tops / MFMA_I8_PEAK_TOPS, 4),
        "check": "every layer: decode(eval labels, garbler zero-labels) = exact integer layer output",
        "layers": layers,
    }


def time_workload(w, steps: int, warmup: int, dev, values: str = "values uniform over the signed range"):
    """Garble, encode and time the evaluator on one workload (HIP events over
    `steps` calls); decode and check every gadget afterwards.  Returns a
    summary dict."""
    import torch

    from paper_2506_14489_amd import binding as B
    from paper_2506_14489_amd import cost
    from paper_2506_14489_amd import workloads as WL

    n = w.n
    x = layer_values(w) if w.kind in ("conv", "fc") else WL.make_inputs(w)
    params = B.make_params(w.moduli, w.scale_idx, n, w.seed)
    buf = B.Buffers(params, dev)
    stream = torch.cuda.current_stream()
    B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work, stream)
    B.redash_encode(params, torch.from_numpy(x).to(dev), buf.in_zero, buf.offsets, buf.in_labels, stream)
    gc.collect()
    # Warm-up: at least `warmup` calls and at least 50 ms of them.  After the CPU
    # has built a layer's inputs the GPU has been idle and a short call gets
    # faster over its first ~30 repetitions (measured: a 200,704-gadget layer
    # from 0.81 to 0.74 ms per call), so a fixed count of a few calls would time
    # small layers on a GPU that has not come back up to speed.
    t_w, done = time.perf_counter(), 0
    while done < warmup or time.perf_counter() - t_w < 0.05:
        B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work, stream)
        done += 1
        if done % 8 == 0:
            torch.cuda.synchronize()
    # An event recorded behind a still-running kernel is stamped when that kernel
    # starts (measured: 10 calls timed that way take 11 calls' time), so the
    # warm-up calls are waited for before the first event.
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work, stream)
    ev1.record(stream)
    B.redash_decode(params, buf.out_labels, buf.out_zero, buf.offsets, buf.y, buf.bad, stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    ok = int(buf.bad.item()) == 0 and np.array_equal(buf.y.cpu().numpy()[:n], expected_values(w, x))
    del buf
    torch.cuda.empty_cache()
    if not ok:
        log(f"{w.name}: decode check FAILED")
        sys.exit(1)
    tops = cost.ops_per_gadget(w.moduli, w.scale_idx) * n / (ms / 1e3) / 1e12
    gbs = cost.bytes_per_gadget(w.moduli, w.scale_idx) * n / (ms / 1e3) / 1e9
    log(f"{w.name}: eval {ms:.3f} ms per call, {n / (ms / 1e3):.3e} gadgets/s")
    return {
        "workload": f"{w.name}: {n} gadgets, {values}",
        "moduli": list(w.moduli),
        "scale": w.s,
        "gates_per_gadget": len(cost.gates(w.moduli, w.scale_idx)),
        "ms_per_call": round(ms, 4),
        "gadgets_per_s": round(n / (ms / 1e3), 1),
        "alu_frac": round(tops / ALU_PEAK_TOPS, 4),
        "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
        "check": "decode = floor((x + (floor(P/2) mod s))/s) with every label valid, all gadgets",
        "steps": steps,
    }


def time_resnet18(steps: int, warmup: int, dev):
    """The 21 ResNet-18 layers one after another (each layer's activations from
    its own int8 input and weights): sum of gadgets over sum of the per-layer
    evaluation times."""
    from paper_2506_14489_amd import cost
    from paper_2506_14489_amd import workloads as WL

    layers, n_tot, ms_tot, ops_tot = [], 0, 0.0, 0
    for w in WL.RESNET18:
        r = time_workload(w, steps, warmup, dev, values="the layer's exact conv/fc outputs")
        layers.append({"layer": w.name, "gadgets": w.n, "scale": w.s, "ms_per_call": r["ms_per_call"]})
        n_tot += w.n
        ms_tot += r["ms_per_call"]
        ops_tot += cost.ops_per_gadget(w.moduli, w.scale_idx) * w.n
    tops = ops_tot / (ms_tot / 1e3) / 1e12
    log(f"resnet18: {n_tot} gadgets in {ms_tot:.3f} ms over {len(layers)} layers")
    return {
        "gadgets": n_tot,
        "ms_total": round(ms_tot, 4),
        "gadgets_per_s": round(n_tot / (ms_tot / 1e3), 1),
        "alu_frac": round(tops / ALU_PEAK_TOPS, 4),
        "check": "every layer: decode = floor((x + (floor(P/2) mod s))/s) with every label valid",
        "layers": layers,
    }


def aes_rate(dev, bitsliced: bool = False, count: int = 1 << 28, reps: int = 5) -> float:
    """AES blocks/s of a bare AES kernel (counter mode under the hash key):
    the evaluator's two-table LDS round code, four blocks per lane, or the
    bitsliced AES, 32 blocks per lane."""
    import torch

    from paper_2506_14489_amd import binding as B

    run = B.redash_aes_ctr_bitsliced if bitsliced else B.redash_aes_ctr
    out = torch.empty(4 * count, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    run(count, 0, out, stream)
    torch.cuda.synchronize()  # (see time_workload: no event behind a running kernel)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        run(count, 0, out, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del out
    torch.cuda.empty_cache()
    log(f"aes ({'bitsliced' if bitsliced else 'round tables'}): {count} blocks in {ms:.3f} ms, "
        f"{count / (ms / 1e3):.3e} blocks/s")
    return count / (ms / 1e3)


def copy_bandwidth(dev, mib: int = 2048, reps: int = 5) -> float:
    """GB/s of a device-to-device copy (bytes read + bytes written)."""
    import torch

    src = torch.ones(mib * (1 << 20) // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * src.numel() * 4 * reps / (e0.elapsed_time(e1) / 1e3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="batched")
    ap.add_argument("--cpu-sample", type=int, default=1024)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cpu-slices", action="store_true", help="time the oracle on the benchmark workload only")
    ap.add_argument("--no-check", action="store_true", help="skip the decode check after timing")
    ap.add_argument("--garble-steps", type=int, default=3,
                    help="timed garbler calls (offline phase, reported beside the evaluator; 0 skips)")
    ap.add_argument("--no-linear", action="store_true",
                    help="skip timing the garbled conv layer that produces the workload's activations "
                         "(and the ResNet-18 linear layers)")
    ap.add_argument("--no-resnet18", action="store_true",
                    help="skip timing the 21 ResNet-18 layers (sum of gadgets over sum of per-layer times)")
    ap.add_argument("--no-short-bases", action="store_true",
                    help="skip timing the evaluator on the short and power-of-two bases of Sec. 4")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 3 device-to-device copies of MIB MiB (reference for HBM byte counters)")
    args = ap.parse_args()

    # The garbage collector runs only where gc.collect() is called, outside
    # timed regions: a collection while short calls are being queued would
    # leave the GPU idle inside the timed interval.
    gc.disable()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(gadgets are independent: a multi-GPU run would shard them, see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n_words = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n_words, dtype=torch.int32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {args.copy_calibration} MiB three times")
        return

    from paper_2506_14489_amd import binding as B
    from paper_2506_14489_amd import cost
    from paper_2506_14489_amd import traffic
    from paper_2506_14489_amd import workloads as WL

    w = WL.by_name(args.workload)
    n = w.n
    log(f"workload {w.name}: {n} gadgets, moduli {w.moduli}, s = {w.s}, seed {w.seed}")
    t0 = time.time()
    x = layer_values(w) if w.kind in ("conv", "fc") else WL.make_inputs(w)
    log(f"inputs ready in {time.time() - t0:.1f} s")

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    params = B.make_params(w.moduli, w.scale_idx, n, w.seed)
    buf = B.Buffers(params, dev)
    stream = torch.cuda.current_stream()
    t0 = time.time()
    B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work, stream)
    xd = torch.from_numpy(x).to(dev)
    B.redash_encode(params, xd, buf.in_zero, buf.offsets, buf.in_labels, stream)
    torch.cuda.synchronize()
    log(f"garbled and encoded on the GPU in {time.time() - t0:.1f} s "
        f"({buf.sizes['table_words'] * 4 / 1e9:.1f} GB of tables)")

    garble = None
    if args.garble_steps > 0:
        # The offline phase on the same buffers (deterministic: rewrites the same tables).
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(args.garble_steps):
            B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work, stream)
        g1.record(stream)
        torch.cuda.synchronize()
        g_ms = g0.elapsed_time(g1) / args.garble_steps
        g_aes = cost.garble_aes_blocks_per_gadget(w.moduli, w.scale_idx)
        g_ops = cost.garble_ops_per_gadget(w.moduli, w.scale_idx)
        g_bytes = cost.garble_bytes_per_gadget(w.moduli, w.scale_idx)
        g_tops = g_ops * n / (g_ms / 1e3) / 1e12
        garble = {
            "ms_per_call": round(g_ms, 3),
            "gadgets_per_s": round(n / (g_ms / 1e3), 1),
            "aes_blocks_per_s": round(g_aes * n / (g_ms / 1e3), 1),
            "table_write_gbs": round(buf.sizes["table_words"] * 4 / (g_ms / 1e3) / 1e9, 1),
            "roofline": {"bound": "alu", "achieved": round(g_tops, 3), "peak": round(ALU_PEAK_TOPS, 2),
                         "unit": "TOP/s", "frac": round(g_tops / ALU_PEAK_TOPS, 4), "ops_per_gadget": g_ops,
                         "kernel": "k_garble"},
            "hbm": {"achieved": round(g_bytes * n / (g_ms / 1e3) / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "bytes_per_gadget": g_bytes},
            "steps": args.garble_steps,
        }
        log(f"garble: {g_ms:.3f} ms per call")

    gc.collect()
    for _ in range(args.warmup):
        B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work, stream)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / args.steps
    log(f"eval: {ms_step:.3f} ms per call (events), wall {wall * 1e3 / args.steps:.3f} ms per call")
    # the same number of calls again, each between its own pair of events: the median call
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for e0, e1 in evs:
        e0.record(stream)
        B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work, stream)
        e1.record(stream)
    torch.cuda.synchronize()
    ms_median = float(np.median([e0.elapsed_time(e1) for e0, e1 in evs]))
    log(f"eval: median {ms_median:.3f} ms per call over {args.steps} separately timed calls")

    check = "skipped"
    if not args.no_check:
        B.redash_decode(params, buf.out_labels, buf.out_zero, buf.offsets, buf.y, buf.bad, stream)
        torch.cuda.synchronize()
        ok = int(buf.bad.item()) == 0 and np.array_equal(buf.y.cpu().numpy()[:n], expected_values(w, x))
        if not ok:
            log("decode check FAILED")
            sys.exit(1)
        check = f"decode = floor(x/s) with every label valid, all {n} gadgets"
        log(check)

    gadgets_per_s = n / (ms_step / 1e3)
    copy_gbs = copy_bandwidth(dev)
    log(f"device-to-device copy: {copy_gbs:.1f} GB/s (read + write)")
    aes_peak = aes_rate(dev)
    aes_bs = aes_rate(dev, bitsliced=True)
    bytes_g = cost.bytes_per_gadget(w.moduli, w.scale_idx)
    ops_g = cost.ops_per_gadget(w.moduli, w.scale_idx)
    lds_g = cost.lds_bytes_per_gadget(w.moduli, w.scale_idx)
    aes_g = cost.aes_blocks_per_gadget(w.moduli, w.scale_idx)
    achieved_tops = ops_g * n / (ms_step / 1e3) / 1e12
    achieved_gbs = bytes_g * n / (ms_step / 1e3) / 1e9
    # HBM bytes per launch from the rocprofv3 counters (None once the kernel changed)
    traffic_b = traffic.traffic_bytes(w.name)
    valu_i = traffic.valu_instructions(w.name)
    result = {
        "metric": METRIC,
        "value": round(gadgets_per_s, 1),
        "unit": "gadgets/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: {n} gadgets" + (f" ({'x'.join(map(str, w.out_shape[1:] if w.out_shape[0] == 1 else w.out_shape))} map)" if w.out_shape else ""),
            "moduli": list(w.moduli),
            "scale": w.s,
            "seed": w.seed,
            "gates_per_gadget": len(cost.gates(w.moduli, w.scale_idx)),
            "aes_blocks_per_gadget": aes_g,
        },
        "roofline": {
            "bound": "alu",
            "achieved": round(achieved_tops, 3),
            "peak": round(ALU_PEAK_TOPS, 2),
            "unit": "TOP/s",
            "frac": round(achieved_tops / ALU_PEAK_TOPS, 4),
            "traffic": traffic_b,
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE x2 + WRITE_SIZE x1)",
            "kernel": "k_eval",
            "ops_per_gadget": ops_g,
        },
        "hbm": {
            "achieved": round(achieved_gbs, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved_gbs / HBM_PEAK_GBS, 4),
            "bytes_per_gadget": round(bytes_g, 1),
            "measured_bytes_per_gadget": None if traffic_b is None else round(traffic_b / n, 1),
            "copy_gbs": round(copy_gbs, 1),
            "frac_of_copy": round(achieved_gbs / copy_gbs, 4),
        },
        "lds": {
            "achieved": round(lds_g * n / (ms_step / 1e3) / 1e9, 1),
            "peak": round(LDS_PEAK_GBS, 1),
            "unit": "GB/s",
            "frac": round(lds_g * n / (ms_step / 1e3) / 1e9 / LDS_PEAK_GBS, 4),
            "bytes_per_gadget": lds_g,
        },
        # measured VALU issue: SQ_INSTS_VALU x 4 cycles per wave64 instruction on a 16-lane SIMD,
        # against 1,024 SIMDs x 2.4 GHz over the launch (None once the kernel changed)
        "valu_issue": {"instructions_per_launch": valu_i,
                       "frac": None if valu_i is None else round(valu_i * 4 / (1024 * 2.4e9 * ms_step / 1e3), 4),
                       "source": "rocprofv3 SQ_INSTS_VALU"},
        "aes_blocks_per_s": round(aes_g * gadgets_per_s, 1),
        "aes_roofline": {"achieved": round(aes_g * gadgets_per_s, 1), "peak": round(aes_peak, 1),
                         "unit": "AES blocks/s", "frac": round(aes_g * gadgets_per_s / aes_peak, 4),
                         "kernel": "k_eval",
                         "peak_kernel": "k_aes_ctr: the evaluator's AES alone (two-table LDS rounds, "
                                        "four blocks per lane, counter mode)",
                         "bitsliced_blocks_per_s": round(aes_bs, 1),
                         "bitsliced_kernel": "k_aes_ctr_bs: bitsliced AES, 32 blocks per lane, Boyar-Peralta "
                                             "S-box, counter mode"},
        "ms_median_per_call": round(ms_median, 4),
        "check": check,
        "garble": garble,
    }
    if not args.no_linear and w.kind == "conv":
        result["linear"] = time_linear_layer(w, params, buf, args.steps, args.warmup, dev)
    del buf
    torch.cuda.empty_cache()
    if not args.no_short_bases:
        # the short and power-of-two bases of Sec. 4, at the batched map's gadget count
        result["short_bases"] = [time_workload(WL.at_size(sw, WL.BATCHED.n), max(args.steps // 2, 1),
                                               args.warmup, dev) for sw in WL.SHORT_BASES]
    if not args.no_resnet18:
        result["resnet18"] = time_resnet18(max(args.steps // 2, 1), args.warmup, dev)
    if not args.no_linear and not args.no_resnet18:
        result["resnet18_linear"] = time_resnet18_linear(max(args.steps // 2, 1), args.warmup, dev)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, x, min(args.cpu_sample, n), args.cpu_seconds,
                                              slices=not args.no_cpu_slices)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
