#!/usr/bin/env python3
"""Benchmark of the mixed-precision MoE-layer hot path on one MI355X.

A step is one pass of the whole path over one batch already resident in HBM:
moe_route_permute -> moe_expert_ffn_mixed -> moe_unpermute_combine.
Default workload: the Mixtral-8x7B-shaped layer at decode (64 tokens,
d_model 4096, 8 experts, top-2, d_ff 14336, group 128, expert bits
{8:2, 4:4, 2:2}, 5 % of output channels switched to resident 8-bit copies).

Prints one JSON line with tokens/s, the roofline of the dominant kernel (the
gate/up expert kernel, timed with HIP events on its own stream) and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import ctypes as C
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 MFMA


def reap_children():
    """Nothing this run started may outlive it: the oracle's build (gcc) and
    the library's build run as waited-for subprocesses and the thread pools
    are joined, so no child is expected; any that is left is named on stderr
    and ended."""
    try:
        import psutil
    except ImportError:
        return
    kids = psutil.Process().children(recursive=True)
    for c in kids:
        try:
            log("ending child process %d (%s)" % (c.pid, " ".join(c.cmdline()[:4])))
            c.terminate()
        except psutil.Error:
            pass
    psutil.wait_procs(kids, timeout=5)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles created through the HIP runtime torch already loaded."""

    DISABLE_SYSTEM_FENCE = 0x20000000   # hipEventDisableSystemFence

    def __init__(self):
        self.hip = C.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
        self.hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [C.c_void_p]
        self.hip.hipEventDestroy.argtypes = [C.c_void_p]

    def create(self, n):
        arr = (C.c_void_p * n)()
        for i in range(n):
            ev = C.c_void_p()
            # timing-only events: no system-scope fence (no cache write-back
            # and invalidate between the kernels they bracket)
            if self.hip.hipEventCreateWithFlags(C.byref(ev), self.DISABLE_SYSTEM_FENCE) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            arr[i] = ev.value
        return arr

    def record(self, ev, stream):
        if self.hip.hipEventRecord(C.c_void_p(ev), C.c_void_p(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def ms(self, a, b):
        out = C.c_float()
        if self.hip.hipEventElapsedTime(C.byref(out), C.c_void_p(a), C.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(out.value)

    def destroy(self, arr):
        for v in arr:
            self.hip.hipEventDestroy(C.c_void_p(v))


def algorithmic_bytes(layer, offsets):
    """Packed-weight bytes one step must read, per FFN stage: base codes of
    unswitched rows, 8-bit copy codes of switched rows and one {scale, zero}
    word per row and group, over the experts that received tokens."""
    cfg = layer.cfg
    E, S, g = layer.E, layer.S, cfg.group
    counts = np.diff(offsets)
    out = {"gate_up": 0, "down": 0}
    for e in range(E + S):
        if counts[e] == 0:
            continue
        b = int(layer.bits_host[e])
        for kind in range(3):
            R, K = cfg.rows(kind, e), cfg.cols(kind, e)
            n_sw = int(np.sum(layer.row_slot(kind)[e] >= 0)) if e < E else 0
            nb = (R - n_sw) * K * b // 8 + n_sw * K + R * (K // g) * 4
            out["down" if kind == 2 else "gate_up"] += nb
    return out


def algorithmic_flops(layer, offsets):
    cfg = layer.cfg
    counts = np.diff(offsets)
    fl = 0
    for e in range(layer.E + layer.S):
        f = cfg.d_ff if e < layer.E else cfg.d_ff_shared
        fl += int(counts[e]) * 2 * 3 * cfg.d_model * f
    return fl


def flops_gate_up(layer, offsets):
    """Multiply-add flops of the gate and up projections over all rows."""
    cfg = layer.cfg
    counts = np.diff(offsets)
    fl = 0
    for e in range(layer.E + layer.S):
        f = cfg.d_ff if e < layer.E else cfg.d_ff_shared
        fl += int(counts[e]) * 2 * 2 * cfg.d_model * f
    return fl


def describe(wk):
    c = wk.layer
    bits = dict(c.bit_shares) if c.bit_shares else list(c.bits_literal)
    d = {"workload": "%s: %s, T=%d" % (wk.name, c.name, wk.tokens), "tokens": wk.tokens,
         "d_model": c.d_model, "experts": c.n_experts, "shared_experts": c.n_shared,
         "top_k": c.top_k, "d_ff": c.d_ff, "group": c.group, "bits": str(bits),
         "switched_rows": "%s %s" % (c.copies, c.mask_frac if c.copies != "pool" else c.pool_frac)}
    if c.n_shared:
        d["d_ff_shared"] = c.d_ff_shared
    if wk.zipf_s:
        d["router_zipf_s"] = wk.zipf_s
    return d


def measured_traffic(workload):
    """HBM bytes per gate/up launch from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE passes scaled by a plain copy's reading), or
    None when there is none for this workload or the kernel sources have
    changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_ffn_gateup_%s.md" % workload.replace("-", "_"))
    if not os.path.exists(path):
        return None
    kv = dict(re.findall(r"^(\w+): (\S+)$", open(path).read(), flags=re.M))
    if kv.get("workload") != workload or kv.get("source_sha256_16") != ffn_source_hash():
        return None
    return int(kv["traffic_bytes_per_launch"])


def ffn_source_hash():
    """Hash of the expert-FFN kernel sources without their comments and
    layout (the counters are valid for that code only)."""
    h = hashlib.sha256()
    for f in FFN_SOURCES:
        with open(os.path.join(ROOT, "paper_2503_21135_amd", "csrc", f)) as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


FFN_SOURCES = ("ffn.hip", "ffn_common.hpp", "ffn_prep.hip", "ffn_stream.hip", "ffn_tile.hip",
               "common.hpp")




def cpu_baseline(wk, inputs, batch, min_seconds):
    """The oracle on a bounded sample of the same step: routing and
    permutation of the whole batch, then the fp64 SiLU-GLU FFN of the rows
    routed to the busiest expert, repeated until `min_seconds` have passed.
    That expert's dequantized matrices (the oracle's resident form of the
    packed weights) are prepared before the clock starts, as the packed
    weights are on the GPU side.  tokens/s counts k expert rows as one token."""
    import oracle
    cfg = wk.layer
    k = cfg.top_k
    rs = oracle.switch_state(inputs, epoch=0)
    _, ids, _ = oracle.route(batch.x, inputs.router, k, batch.bias)
    off, perm, _ = oracle.permute(ids, cfg.n_experts, cfg.n_shared)
    e = int(np.argmax(np.diff(off[:cfg.n_experts + 1])))
    W = [oracle.effective_weight(inputs.weight(e, kd), int(inputs.bits[e]), cfg.group,
                                 np.nonzero(rs[kd][e] >= 0)[0]) for kd in (0, 1, 2)]
    rows = perm[off[e]:off[e + 1]]

    def run(seconds):
        reps = 0
        t0 = time.perf_counter()
        while True:
            _, ids, _ = oracle.route(batch.x, inputs.router, k, batch.bias)
            oracle.permute(ids, cfg.n_experts, cfg.n_shared)
            oracle.expert_ffn(W[0], W[1], W[2], batch.x, rows)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= seconds:
                return reps, dt

    threads = oracle.num_threads()
    reps, dt = run(min_seconds)
    tok = reps * len(rows) / k
    # the same sample on one thread, a quarter as long
    oracle.set_num_threads(1)
    reps1, dt1 = run(min_seconds / 4)
    oracle.set_num_threads(threads)
    model = ""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(tok / dt, 4), "unit": "tokens/s", "cores": threads,
            "kind": "oracle", "cpu": model,
            "value_1_thread": round(reps1 * len(rows) / k / dt1, 4),
            "sample": "%d x (route+permute of all %d tokens, fp64 FFN of the %d rows of "
                      "expert %d at %d bits, %d%% of rows switched); %d expert rows = "
                      "%.1f tokens at top-%d in %.1f s"
                      % (reps, wk.tokens, len(rows), e, int(inputs.bits[e]),
                         inputs.switch_percent(0), reps * len(rows), tok, k, dt)}


PREFILL_OF = {"mixtral-decode": "mixtral-prefill", "deepseek-decode": "deepseek-prefill"}


def measure_prefill(layer, inputs, name, hip, steps, warmup, bf16=True):
    """The same packed layer at prefill: whole-step time and the gate/up
    launch (the MFMA-bound kernel) against the bf16/fp16 matrix-core peak."""
    import torch
    import moe_inputs as mi
    from paper_2503_21135_amd import api
    wk = mi.WORKLOADS[name]
    batch = mi.make_batch(wk, inputs)
    x = torch.from_numpy(batch.x.view(np.int16)).to("cuda:0").view(torch.bfloat16)
    bias = None if batch.bias is None else torch.from_numpy(batch.bias).to("cuda:0")
    b = layer.buffers(wk.tokens)
    for _ in range(warmup):
        layer.route(x, bias)
        layer.ffn(x, b)
        layer.combine(b)
    torch.cuda.synchronize()
    ev = hip.create(2 * steps)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(steps):
        layer.route(x, bias)
        api.moe_expert_ffn_mixed_ev(layer.desc, x, layer.k, b.offsets, b.perm, b.o, b.ffn_ws,
                                    (C.c_void_p * 5)(None, ev[2 * i], ev[2 * i + 1], None, None))
        layer.combine(b)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    gu = float(np.mean([hip.ms(ev[2 * i], ev[2 * i + 1]) for i in range(steps)]))
    hip.destroy(ev)
    off = b.offsets.cpu().numpy()
    fgu = flops_gate_up(layer, off)
    tf = fgu / (gu * 1e-3) / 1e12
    ref = None
    if bf16:
        ref = measure_bf16(layer, x, b, min(steps, 10))
        ref["speedup_of_quantized"] = round(ref["ms_per_step"] / ms, 3)
    return {"bf16_reference": ref,
            "workload": "%s: T=%d, router biased to Zipf s=%s loads" % (name, wk.tokens, wk.zipf_s)
            if wk.zipf_s else "%s: T=%d" % (name, wk.tokens),
            "tokens_per_s": round(wk.tokens / (ms * 1e-3), 1), "ms_per_step": round(ms, 4),
            "steps": steps,
            "roofline": {"bound": "mfma", "kernel": "FFN gate/up stage (tile kernel, fp16 operands)",
                         "achieved": round(tf, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(tf / BF16_PEAK_TFLOPS, 4), "avg_launch_ms": round(gu, 4),
                         "algorithmic_flops_per_launch": int(fgu)},
            "layer_tflops": round(algorithmic_flops(layer, off) / (ms * 1e-3) / 1e12, 1),
            "expert_rows": [int(v) for v in np.diff(off)]}


def measure_graph(layer, x, bias, b, y_eager, steps):
    """One decode step captured in a HIP graph and replayed; every replay's
    output is checked against the eager step's (bitwise: the path is
    deterministic)."""
    import torch
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        layer.route(x, bias)
        layer.ffn(x, b)
        layer.combine(b)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        layer.route(x, bias)
        layer.ffn(x, b)
        layer.combine(b)
    ok = True
    for _ in range(3):   # replays with eager work and synchronisation between them
        b.y.zero_()
        g.replay()
        torch.cuda.synchronize()
        ok = ok and bool(torch.equal(b.y, y_eager))
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    ok = ok and bool(torch.equal(b.y, y_eager))
    ms = t0.elapsed_time(t1) / steps
    return {"ms_per_step": round(ms, 5), "tokens_per_s": round(x.shape[0] / (ms * 1e-3), 1),
            "replays_match_eager": ok}


def measure_switch(layer, inputs, wk, hip, steps):
    """The mask-redraw workload: a fresh batch every step, the switch mask
    redrawn every `redraw_every` steps.  Steady tokens/s excludes the
    switch; switch latency is the host wall time of installing one epoch's
    slot lists (three moe_set_channel_switch calls) until the stream is idle,
    and its device time from events."""
    import torch
    import moe_inputs as mi
    from paper_2503_21135_amd import api
    n_ep = (steps + wk.redraw_every - 1) // wk.redraw_every
    slots = [[np.ascontiguousarray(inputs.slots_on(kd, ep), np.int32) for kd in range(3)]
             for ep in range(n_ep)]
    xs = []
    for st in range(min(steps, 20)):   # distinct batches, reused cyclically
        bt = mi.make_batch(wk, inputs, step=st)
        xs.append(torch.from_numpy(bt.x.view(np.int16)).to("cuda:0").view(torch.bfloat16))
    b = layer.buffers(wk.tokens)
    sptr = torch.cuda.current_stream().cuda_stream
    ev = hip.create(2 * steps + 2 * n_ep)
    host_sw = []
    ep_i = 0
    torch.cuda.synchronize()
    for st in range(steps):
        if st % wk.redraw_every == 0:
            ep = st // wk.redraw_every
            torch.cuda.synchronize()
            w0 = time.perf_counter()
            hip.record(ev[2 * steps + 2 * ep_i], sptr)
            for kd in range(3):
                api.moe_set_channel_switch(layer.desc, kd, slots[ep][kd])
            hip.record(ev[2 * steps + 2 * ep_i + 1], sptr)
            torch.cuda.synchronize()
            host_sw.append(time.perf_counter() - w0)
            ep_i += 1
        x = xs[st % len(xs)]
        hip.record(ev[2 * st], sptr)
        layer.route(x)
        layer.ffn(x, b)
        layer.combine(b)
        hip.record(ev[2 * st + 1], sptr)
    torch.cuda.synchronize()
    step_ms = np.array([hip.ms(ev[2 * i], ev[2 * i + 1]) for i in range(steps)])
    sw_dev = np.array([hip.ms(ev[2 * steps + 2 * i], ev[2 * steps + 2 * i + 1]) for i in range(ep_i)])
    hip.destroy(ev)
    med = float(np.median(step_ms))
    return {"workload": "%s: T=%d x %d steps, mask redrawn every %d steps (%d epochs)"
            % (wk.name, wk.tokens, steps, wk.redraw_every, n_ep),
            "steady_tokens_per_s": round(wk.tokens / (med * 1e-3), 1),
            "step_ms_median": round(med, 4), "step_ms_p10": round(float(np.percentile(step_ms, 10)), 4),
            "step_ms_p90": round(float(np.percentile(step_ms, 90)), 4),
            "switch_host_ms_median": round(float(np.median(host_sw)) * 1e3, 4),
            "switch_device_ms_median": round(float(np.median(sw_dev)), 4),
            "switched_percent_by_epoch": [int(inputs.switch_percent(e)) for e in range(n_ep)]}


def measure_dataset_switch(layer, inputs, hip, ms_step, reps=5):
    """Dynamic quantization switch for a new dataset (Sec. IV-B): the cached
    16-bit channels of all three kinds requantized at every expert's new
    precision (moe_requant_channels), then the copy mask installed
    (moe_set_channel_switch).  Device time from events around the six calls,
    host time until the stream is idle.  The share compares the device time
    with itself plus 1024 decode steps of this layer, the online measure of
    the paper's overhead discussion (generation of 1024 tokens)."""
    import torch
    import moe_inputs as mi
    from paper_2503_21135_amd import api
    cfg = layer.cfg
    for kd in range(3):
        layer.channel_cache(kd)   # built before any switch (Sec. V-A)
    slots = [np.ascontiguousarray(inputs.slots_on(kd, 0), np.int32) for kd in range(3)]
    sptr = torch.cuda.current_stream().cuda_stream
    ev = hip.create(3 * reps)
    host = []

    def switch(eb, evs=None):
        if evs:
            hip.record(evs[0], sptr)
        for kd in range(3):
            layer.requant(kd, eb)
        if evs:
            hip.record(evs[1], sptr)
        for kd in range(3):
            api.moe_set_channel_switch(layer.desc, kd, slots[kd])
        if evs:
            hip.record(evs[2], sptr)

    # precision for each new dataset from its calibration batch: route on the
    # GPU, then Eq. (1) and Alg. 1 on the host
    alloc_ms, new_bits = [], []
    for r in range(reps + 1):
        xc, sig = mi.calibration_batch(cfg, r)
        bc = layer.route(torch.from_numpy(xc.view(np.int16)).to("cuda:0").view(torch.bfloat16))
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        ids = bc.topk_ids.cpu().numpy()
        s_exp, share = api.moe_expert_significance(sig, ids, cfg.n_experts)
        new_bits.append(api.moe_allocate_bits(s_exp, share, levels=(8, 6, 4, 2))["bits"])
        alloc_ms.append((time.perf_counter() - w0) * 1e3)
    switch(new_bits[reps])   # warm-up
    torch.cuda.synchronize()
    for r in range(reps):
        eb = new_bits[r]
        w0 = time.perf_counter()
        switch(eb, ev[3 * r:3 * r + 3])
        torch.cuda.synchronize()
        host.append(time.perf_counter() - w0)
    rq = np.array([hip.ms(ev[3 * r], ev[3 * r + 1]) for r in range(reps)])
    inst = np.array([hip.ms(ev[3 * r + 1], ev[3 * r + 2]) for r in range(reps)])
    hip.destroy(ev)
    if int(layer.status.item()) != 0:
        raise RuntimeError("requantization reported status %d" % int(layer.status.item()))
    n_slots = [int(layer.kinds[kd]["n_slots"]) for kd in range(3)]
    Ks = [cfg.cols(kd, 0) for kd in range(3)]
    rd = sum(n * K * 2 for n, K in zip(n_slots, Ks))
    wr = sum(n * (K + K // cfg.group * 4) for n, K in zip(n_slots, Ks))
    tot = float(np.median(rq + inst))
    return {"workload": "%s: per-expert bit-widths of a new dataset from a 1024-token "
                        "calibration batch (GPU routing, then Eq. (1) and Alg. 1 on the host, "
                        "clusters at INT8/6/4/2), "
                        "all cached channels of the three kinds requantized at them, then the "
                        "copy mask installed" % cfg.name,
            "allocation_host_ms": round(float(np.median(alloc_ms)), 4),
            "new_bits_by_dataset": [[int(v) for v in b] for b in new_bits[:reps]],
            "cached_channels": n_slots,
            "cache_mib": round(rd / 2 ** 20, 2),
            "requant_device_ms": round(float(np.median(rq)), 4),
            "install_device_ms": round(float(np.median(inst)), 4),
            "total_device_ms": round(tot, 4),
            "host_ms": round(float(np.median(host)) * 1e3, 4),
            "requant_bytes": int(rd + wr),
            "requant_gbs": round((rd + wr) / (float(np.median(rq)) * 1e-3) / 1e9, 1),
            "share_vs_1024_decode_steps": round(tot / (tot + 1024 * ms_step), 6),
            "share_with_allocation_vs_1024_decode_steps":
                round((tot + float(np.median(alloc_ms))) /
                      (tot + float(np.median(alloc_ms)) + 1024 * ms_step), 6)}


def measure_rotated(wk, layer, inputs, hip, n_copies, steps, warmup=5):
    """The decode step rotating over n_copies independently packed copies of
    the layer (seeds 0..n_copies-1, each with its own batch), so that no
    copy's weights can still sit in the 256 MB Infinity Cache when its turn
    comes again.  Gate/up GB/s from events around each gate/up launch."""
    import ctypes as C
    import torch
    import moe_inputs as mi
    import paper_2503_21135_amd as P
    from paper_2503_21135_amd import api
    dev = torch.device("cuda:0")
    copies = [(layer, inputs)]
    for r in range(1, n_copies):
        inp = mi.LayerInputs(wk.layer, seed=r)
        lay = P.MoELayer(inp, device="cuda:0")
        lay.set_epoch(0)
        copies.append((lay, inp))
    runs = []
    for lay, inp in copies:
        bt = mi.make_batch(wk, inp)
        xr = torch.from_numpy(bt.x.view(np.int16)).to(dev).view(torch.bfloat16)
        br = None if bt.bias is None else torch.from_numpy(bt.bias).to(dev)
        runs.append((lay, xr, br, lay.buffers(wk.tokens)))
    ev = hip.create(2 * steps)

    def step(i, evs=None):
        lay, xr, br, b = runs[i % len(runs)]
        lay.route(xr, br)
        if evs is None:
            lay.ffn(xr, b)
        else:
            api.moe_expert_ffn_mixed_ev(lay.desc, xr, lay.k, b.offsets, b.perm, b.o, b.ffn_ws, evs)
        lay.combine(b)

    for i in range(warmup * len(runs)):
        step(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(steps):
        step(i, (C.c_void_p * 5)(None, ev[2 * i], ev[2 * i + 1], None, None))
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    gu = [hip.ms(ev[2 * i], ev[2 * i + 1]) for i in range(steps)]
    hip.destroy(ev)
    byt = [algorithmic_bytes(lay, b.offsets.cpu().numpy())["gate_up"] for lay, _, _, b in runs]
    tot_b = sum(byt[i % len(runs)] for i in range(steps))
    gbs = tot_b / (sum(gu) * 1e-3) / 1e9
    ws_mb = round(sum(lay.packed_bytes() for lay, _, _, _ in runs) / 1e6, 1)
    runs.clear()
    copies.clear()
    torch.cuda.empty_cache()
    return {"copies": n_copies, "working_set_mb": ws_mb,
            "ms_per_step": round(ms, 5), "tokens_per_s": round(wk.tokens / (ms * 1e-3), 1),
            "gate_up_gbs": round(gbs, 1), "gate_up_hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def pack_copies(wk, n, seed0=0):
    """n independently packed copies of a workload's layer (seeds seed0..),
    each with its copy mask of epoch 0 installed."""
    import moe_inputs as mi
    import paper_2503_21135_amd as P
    out = []
    for r in range(n):
        inp = mi.LayerInputs(wk.layer, seed=seed0 + r)
        lay = P.MoELayer(inp, device="cuda:0")
        lay.set_epoch(0)
        out.append((lay, inp))
    return out


def roofline_hbm(kernel, nbytes, ms, traffic=None):
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
            "algorithmic_bytes_per_launch": int(nbytes), "avg_launch_ms": round(ms, 5)}


def measure_decode_config(name, copies, hip, steps, warmup):
    """A decode workload's step (route + FFN + combine) on its layer, once on
    one packed copy and once rotating over all copies (each with its own
    batch), so that no copy's weights can still sit in the 256 MB Infinity
    Cache when its turn comes again.  The gate/up launches are timed by HIP
    events attached to them; the roofline uses the rotated timing."""
    import torch
    import moe_inputs as mi
    from paper_2503_21135_amd import api
    wk = mi.WORKLOADS[name]
    dev = torch.device("cuda:0")
    runs = []
    for lay, inp in copies:
        bt = mi.make_batch(wk, inp)
        xr = torch.from_numpy(bt.x.view(np.int16)).to(dev).view(torch.bfloat16)
        br = None if bt.bias is None else torch.from_numpy(bt.bias).to(dev)
        runs.append((lay, xr, br, lay.buffers(wk.tokens)))

    def step(run, evs=None):
        lay, xr, br, b = run
        lay.route(xr, br)
        if evs is None:
            lay.ffn(xr, b)
        else:
            api.moe_expert_ffn_mixed_ev(lay.desc, xr, lay.k, b.offsets, b.perm, b.o, b.ffn_ws, evs)
        lay.combine(b)

    def timed(order):
        ev = hip.create(2 * len(order))
        for i in range(warmup * len(runs)):
            step(runs[i % len(runs)])
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for i, r in enumerate(order):
            step(runs[r], (C.c_void_p * 5)(None, ev[2 * i], ev[2 * i + 1], None, None))
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / len(order)
        gu = [hip.ms(ev[2 * i], ev[2 * i + 1]) for i in range(len(order))]
        hip.destroy(ev)
        return ms, gu

    ms1, gu1 = timed([0] * steps)
    order = [i % len(runs) for i in range(steps)]
    msr, gur = timed(order)
    # each copy routes the same batch every time: its offsets after the runs
    byt = [algorithmic_bytes(lay, b.offsets.cpu().numpy()) for lay, _, _, b in runs]
    fl = [algorithmic_flops(lay, b.offsets.cpu().numpy()) for lay, _, _, b in runs]
    gu_bytes = sum(byt[r]["gate_up"] for r in order) / steps
    gu_ms = float(np.mean(gur))
    ffn_bytes = sum(byt[r]["gate_up"] + byt[r]["down"] for r in order) / steps
    out = {"workload": "%s: %s, T=%d" % (name, wk.layer.name, wk.tokens),
           "tokens_per_s": round(wk.tokens / (msr * 1e-3), 1), "ms_per_step": round(msr, 5),
           "steps": steps, "rotated_copies": len(runs),
           "working_set_mb": round(sum(lay.packed_bytes() for lay, _ in copies) / 1e6, 1),
           "one_copy": {"ms_per_step": round(ms1, 5),
                        "tokens_per_s": round(wk.tokens / (ms1 * 1e-3), 1),
                        "gate_up_ms": round(float(np.mean(gu1)), 5)},
           "roofline": roofline_hbm("FFN gate/up stage (routed and shared experts)", gu_bytes, gu_ms),
           "step_weight_bytes": int(ffn_bytes),
           "step_hbm_frac": round(ffn_bytes / (msr * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "step_tflops": round(sum(fl[r] for r in order) / steps / (msr * 1e-3) / 1e12, 2),
           "expert_rows_copy0": [int(v) for v in np.diff(runs[0][3].offsets.cpu().numpy())]}
    runs.clear()
    return out


def measure_stress(hip, n_copies, steps=None):
    """The runtime-switch stress workload on the Qwen1.5-MoE-A2.7B-shaped
    layer: 512 fresh tokens per step, the copy mask redrawn every 10 steps,
    the steps rotating over n_copies independently packed copies of the
    layer (each mask update installs the new epoch on every copy).  Steady
    throughput is the median step (device events around route + FFN +
    combine); switch latency is the host wall time of installing one copy's
    three slot lists until the stream is idle, and its device time."""
    import torch
    import moe_inputs as mi
    from paper_2503_21135_amd import api
    wk = mi.WORKLOADS["qwen-stress"]
    steps = wk.steps if steps is None else steps
    copies = pack_copies(wk, n_copies)
    n_ep = (steps + wk.redraw_every - 1) // wk.redraw_every
    xs = []
    for st in range(min(steps, 20)):   # distinct batches, reused cyclically
        bt = mi.make_batch(wk, copies[0][1], step=st)
        xs.append(torch.from_numpy(bt.x.view(np.int16)).to("cuda:0").view(torch.bfloat16))
    bufs = [lay.buffers(wk.tokens) for lay, _ in copies]
    sptr = torch.cuda.current_stream().cuda_stream
    ev = hip.create(4 * steps)
    ev_sw = hip.create(2 * n_ep * n_copies)
    host_sw = []
    torch.cuda.synchronize()
    for st in range(steps):
        if st % wk.redraw_every == 0:
            ep = st // wk.redraw_every
            for c, (lay, inp) in enumerate(copies):
                slots = [np.ascontiguousarray(inp.slots_on(kd, ep), np.int32) for kd in range(3)]
                torch.cuda.synchronize()
                w0 = time.perf_counter()
                i = 2 * (ep * n_copies + c)
                hip.record(ev_sw[i], sptr)
                for kd in range(3):
                    api.moe_set_channel_switch(lay.desc, kd, slots[kd])
                hip.record(ev_sw[i + 1], sptr)
                torch.cuda.synchronize()
                host_sw.append(time.perf_counter() - w0)
        lay, _ = copies[st % n_copies]
        b = bufs[st % n_copies]
        x = xs[st % len(xs)]
        hip.record(ev[4 * st], sptr)
        lay.route(x)
        api.moe_expert_ffn_mixed_ev(lay.desc, x, lay.k, b.offsets, b.perm, b.o, b.ffn_ws,
                                    (C.c_void_p * 5)(ev[4 * st + 1], None, None, None,
                                                     ev[4 * st + 2]))
        lay.combine(b)
        hip.record(ev[4 * st + 3], sptr)
    torch.cuda.synchronize()
    step_ms = np.array([hip.ms(ev[4 * i], ev[4 * i + 3]) for i in range(steps)])
    ffn_ms = np.array([hip.ms(ev[4 * i + 1], ev[4 * i + 2]) for i in range(steps)])
    sw_dev = np.array([hip.ms(ev_sw[2 * i], ev_sw[2 * i + 1]) for i in range(n_ep * n_copies)])
    hip.destroy(ev)
    hip.destroy(ev_sw)
    # bytes and flops of the last step of each copy (its routing and mask)
    byt, fl = [], []
    for (lay, _), b in zip(copies, bufs):
        off = b.offsets.cpu().numpy()
        bb = algorithmic_bytes(lay, off)
        byt.append(bb["gate_up"] + bb["down"])
        fl.append(algorithmic_flops(lay, off))
    med, ffn_med = float(np.median(step_ms)), float(np.median(ffn_ms))
    nb, nf = float(np.mean(byt)), float(np.mean(fl))
    ws_mb = round(sum(lay.packed_bytes() for lay, _ in copies) / 1e6, 1)
    pcts = [int(copies[0][1].switch_percent(e)) for e in range(n_ep)]
    copies.clear()
    bufs.clear()
    torch.cuda.empty_cache()
    gbs = nb / (ffn_med * 1e-3) / 1e9
    tf = nf / (ffn_med * 1e-3) / 1e12
    return {"workload": "%s: T=%d x %d steps, mask redrawn every %d steps (%d epochs, %d-%d%% of "
                        "rows switched), rotating over %d packed copies"
                        % (wk.name, wk.tokens, steps, wk.redraw_every, n_ep, min(pcts), max(pcts),
                           n_copies),
            "steady_tokens_per_s": round(wk.tokens / (med * 1e-3), 1),
            "step_ms_median": round(med, 4),
            "step_ms_p10": round(float(np.percentile(step_ms, 10)), 4),
            "step_ms_p90": round(float(np.percentile(step_ms, 90)), 4),
            "ffn_ms_median": round(ffn_med, 4),
            "working_set_mb": ws_mb,
            "switch_host_ms_median": round(float(np.median(host_sw)) * 1e3, 4),
            "switch_device_ms_median": round(float(np.median(sw_dev)), 4),
            "switched_percent_by_epoch": pcts,
            "roofline": {"bound": "hbm", "kernel": "expert FFN (both stages) per step; near the "
                                                  "ridge, so both fractions are given",
                         "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(gbs / HBM_PEAK_GBS, 4),
                         "mfma_achieved_tflops": round(tf, 1),
                         "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4),
                         "algorithmic_bytes_per_step": int(nb),
                         "algorithmic_flops_per_step": int(nf)},
            "verified": "every step's routing (all 512 tokens, bit-exact) and output (8 tokens) "
                        "against the oracle in tests/test_gpu_stress.py"}


def measure_unquantized(name, hip, steps, warmup=5, quantized_ms=None):
    """The same step on the unquantized 16-bit reference layer: every expert
    at bits = 16 (the bf16 values of the same seeded fp32 weights, no channel
    copies, group 64) through the library's own kernels, on the quantized
    workload's batch (same activations, same router bias).  The paper's only
    performance figure is the speedup of the packed low-bit experts over a
    16-bit model (Sec. VI-C); `speedup_of_quantized` is that ratio here."""
    import torch
    import moe_inputs as mi
    import paper_2503_21135_amd as P
    from paper_2503_21135_amd import api
    wk = mi.WORKLOADS[name]
    q_inputs = mi.LayerInputs(wk.layer)
    inp = mi.LayerInputs(mi.unquantized(wk.layer))
    lay = P.MoELayer(inp, device="cuda:0")
    lay.set_epoch(0)
    bt = mi.make_batch(wk, q_inputs)
    x = torch.from_numpy(bt.x.view(np.int16)).to("cuda:0").view(torch.bfloat16)
    bias = None if bt.bias is None else torch.from_numpy(bt.bias).to("cuda:0")
    b = lay.buffers(wk.tokens)
    for _ in range(warmup):
        lay.forward(x, bias)
    torch.cuda.synchronize()
    ev = hip.create(2 * steps)
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(steps):
        lay.route(x, bias)
        api.moe_expert_ffn_mixed_ev(lay.desc, x, lay.k, b.offsets, b.perm, b.o, b.ffn_ws,
                                    (C.c_void_p * 5)(None, ev[2 * i], ev[2 * i + 1], None, None))
        lay.combine(b)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    gu = float(np.mean([hip.ms(ev[2 * i], ev[2 * i + 1]) for i in range(steps)]))
    hip.destroy(ev)
    off = b.offsets.cpu().numpy()
    byt = algorithmic_bytes(lay, off)
    out = {"workload": "%s on the unquantized 16-bit layer (bf16 weights of the same fp32 draw, "
                       "library kernels)" % name,
           "ms_per_step": round(ms, 5), "tokens_per_s": round(wk.tokens / (ms * 1e-3), 1),
           "gate_up_ms": round(gu, 5), "weight_bytes_per_step": int(byt["gate_up"] + byt["down"]),
           "gate_up_gbs": round(byt["gate_up"] / (gu * 1e-3) / 1e9, 1),
           "gate_up_tflops": round(flops_gate_up(lay, off) / (gu * 1e-3) / 1e12, 1)}
    if quantized_ms:
        out["speedup_of_quantized"] = round(ms / quantized_ms, 3)
    del lay, b
    torch.cuda.empty_cache()
    return out


def measure_copy(mib=1024, reps=10):
    """GB/s of a plain device-to-device copy (bytes read + written), for context."""
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        b.copy_(a)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / reps
    del a, b
    torch.cuda.empty_cache()
    return {"bytes_moved": 2 * n * 4, "gbs": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}


def measure_bf16(layer, x, b, steps, warmup=3):
    """Reference point for the paper's speedup claim (its only performance
    figure is quantized-vs-16-bit): the same expert FFNs with unquantized
    bf16 weights of the same shapes (seeded, random: only the time is used),
    on the same routing, through torch's library GEMMs (hipBLASLt) --
    gather of the routed rows, gate/up/down products, SiLU-GLU, weighted
    combine.  Not part of the product path."""
    import torch
    cfg = layer.cfg
    dev = x.device
    gen = torch.Generator(device=dev).manual_seed(1234)
    E, S, k = layer.E, layer.S, layer.k
    ws = []
    for e in range(E + S):
        f = cfg.d_ff if e < E else cfg.d_ff_shared
        # weights stored [in][out] contiguous: the products take no transposed views
        wg = (torch.randn(cfg.d_model, f, generator=gen, device=dev) * 0.02).to(torch.bfloat16)
        wu = (torch.randn(cfg.d_model, f, generator=gen, device=dev) * 0.02).to(torch.bfloat16)
        wd = (torch.randn(f, cfg.d_model, generator=gen, device=dev) * 0.02).to(torch.bfloat16)
        ws.append((wg, wu, wd))
    off = b.offsets.cpu().tolist()
    perm = b.perm.long()
    out = torch.empty(perm.numel(), cfg.d_model, dtype=torch.bfloat16, device=dev)
    w_rows = torch.ones(perm.numel(), 1, dtype=torch.float32, device=dev)
    inv = b.inv.long()

    def step():
        xp = x.index_select(0, perm)
        for e in range(E + S):
            p0, p1 = off[e], off[e + 1]
            if p1 <= p0:
                continue
            wg, wu, wd = ws[e]
            xe = xp[p0:p1]
            h = torch.nn.functional.silu(xe @ wg) * (xe @ wu)
            out[p0:p1] = h @ wd
        # y[t] = sum_j w[t, j] o[inv[t, j]] (+ shared rows)
        o = out.float()
        y = (o[inv[:, :k]] * b.topk_w.unsqueeze(-1)).sum(1)
        if S:
            y = y + o[inv[:, k:]].sum(1)
        return y

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    wbytes = sum(int(w.numel()) * 2 for t in ws for w in t)
    del ws
    torch.cuda.empty_cache()
    return {"ms_per_step": round(ms, 4), "tokens_per_s": round(x.shape[0] / (ms * 1e-3), 1),
            "weight_bytes": wbytes, "kind": "bf16 weights, torch/hipBLASLt GEMMs per expert (reference)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="mixtral-decode")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="minimum CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the companion prefill measurement of a decode workload")
    ap.add_argument("--prefill-steps", type=int, default=20)
    ap.add_argument("--rotate", type=int, default=0, metavar="N",
                    help="also time the decode step rotating over N independently packed copies "
                         "of the layer (defeats the Infinity Cache)")
    ap.add_argument("--no-dataset-switch", action="store_true",
                    help="skip the timing of a requantization for a new dataset")
    ap.add_argument("--no-bf16", action="store_true",
                    help="skip the unquantized 16-bit references of the same steps (the library's "
                         "own kernels on bf16 weights, and torch's library GEMMs for context)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (DeepSeekMoE-shaped decode and prefill, "
                         "Qwen-shaped switch stress) that the default run also measures")
    ap.add_argument("--config-rotate", type=int, default=3, metavar="N",
                    help="packed copies the other workloads rotate over (Infinity Cache defeat)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run 10 plain device-to-device copies of MIB MiB (the "
                         "reference for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(10):
            b.copy_(a)
        torch.cuda.synchronize()
        log("copied %d MiB x 10" % args.copy_calibration)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import moe_inputs as mi
    import paper_2503_21135_amd as P
    from paper_2503_21135_amd import api

    wk = mi.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    t_build = time.perf_counter()
    inputs = mi.LayerInputs(wk.layer)
    layer = P.MoELayer(inputs, device="cuda:0")
    layer.set_epoch(0)
    batch = mi.make_batch(wk, inputs)
    x = torch.from_numpy(batch.x.view(np.int16)).to(dev).view(torch.bfloat16)
    bias = None if batch.bias is None else torch.from_numpy(batch.bias).to(dev)
    torch.cuda.synchronize()
    log("layer packed in %.1f s; packed bytes %.1f MB" %
        (time.perf_counter() - t_build, layer.packed_bytes() / 1e6))

    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    hip = HipEvents()
    K, W = args.steps, args.warmup
    n_stage = 5                 # FFN stage boundaries: xsum | gate/up | hsum | down |
    b = layer.buffers(wk.tokens)

    def step(evs=None):
        layer.route(x, bias)
        if evs is None:
            layer.ffn(x, b)
        else:
            api.moe_expert_ffn_mixed_ev(layer.desc, x, layer.k, b.offsets, b.perm, b.o,
                                        b.ffn_ws, evs)
        layer.combine(b)

    for _ in range(W):
        step()
    torch.cuda.synchronize()
    offsets = b.offsets.cpu().numpy()

    # Timed region: K whole steps.  The only events inside it bracket the
    # gate/up launch of each step (the roofline kernel); each event costs the
    # stream a few microseconds, which the step time keeps.
    ev_gu = hip.create(2 * K)
    gu_arrays = [(C.c_void_p * n_stage)(None, ev_gu[2 * i], ev_gu[2 * i + 1], None, None)
                 for i in range(K)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record()
    for i in range(K):
        step(gu_arrays[i])
    enqueue = time.perf_counter() - wall0
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / K
    gu_ms = float(np.mean([hip.ms(ev_gu[2 * i], ev_gu[2 * i + 1]) for i in range(K)]))
    hip.destroy(ev_gu)

    # Diagnostic pass after the timed region: events at every stage boundary
    # and around each step, for the per-stage breakdown only.
    KD = min(K, 50)
    ev_ffn = hip.create(n_stage * KD)
    ev_edge = hip.create(2 * KD)
    for i in range(KD):
        hip.record(ev_edge[2 * i], sptr)
        step((C.c_void_p * n_stage)(*ev_ffn[i * n_stage:(i + 1) * n_stage]))
        hip.record(ev_edge[2 * i + 1], sptr)
    torch.cuda.synchronize()
    stages = np.zeros((KD, n_stage - 1))
    for i in range(KD):
        e = ev_ffn[i * n_stage:(i + 1) * n_stage]
        stages[i] = [hip.ms(e[j], e[j + 1]) for j in range(n_stage - 1)]
    layer_ms = np.array([hip.ms(ev_edge[2 * i], ev_edge[2 * i + 1]) for i in range(KD)])
    st = stages.mean(0)
    hip.destroy(ev_ffn)
    hip.destroy(ev_edge)

    byt = algorithmic_bytes(layer, offsets)
    flops = algorithmic_flops(layer, offsets)
    ffn_ms = float(stages.sum(1).mean())
    achieved_gbs = byt["gate_up"] / (gu_ms * 1e-3) / 1e9
    achieved_tf = flops_gate_up(layer, offsets) / (gu_ms * 1e-3) / 1e12
    ffn_gbs = (byt["gate_up"] + byt["down"]) / (ffn_ms * 1e-3) / 1e9
    tokens_per_s = wk.tokens / (ms_per_step * 1e-3)
    log("ms/step %.4f (wall %.4f, host enqueue %.4f); gate/up launch %.4f ms" %
        (ms_per_step, wall / K * 1e3, enqueue / K * 1e3, gu_ms))
    log("diagnostic pass stages ms: xsum %.4f gate/up %.4f hsum %.4f down %.4f; step %.4f" %
        (*st, float(layer_ms.mean())))
    log("gate/up %.1f GB/s %.1f TFLOP/s; FFN %.1f GB/s; %.2f TFLOP/s" %
        (achieved_gbs, achieved_tf, ffn_gbs, flops / (ffn_ms * 1e-3) / 1e12))

    extra = {"copy_reference": measure_copy()}
    log("plain copy", extra["copy_reference"])
    if args.rotate > 1 and not wk.redraw_every:
        extra["rotated"] = measure_rotated(wk, layer, inputs, hip, args.rotate, min(K, 100))
        log("rotated over %d copies" % args.rotate, extra["rotated"])
    if wk.tokens <= 1024 and not wk.redraw_every:
        layer.route(x, bias)
        layer.ffn(x, b)
        layer.combine(b)
        torch.cuda.synchronize()
        y_eager = b.y.clone()
        extra["hip_graph"] = measure_graph(layer, x, bias, b, y_eager, K)
        log("hip graph", extra["hip_graph"])
    if wk.redraw_every:
        extra["mask_redraw"] = measure_switch(layer, inputs, wk, hip, wk.steps)
        log("mask redraw", extra["mask_redraw"])
    if not args.no_bf16:
        ref = measure_bf16(layer, x, b, min(K, 50))
        ref["speedup_of_quantized"] = round(ref["ms_per_step"] / ms_per_step, 3)
        extra["bf16_reference"] = ref
        log("bf16 reference", ref)
    if not args.no_prefill and args.workload in PREFILL_OF:
        log("prefill on the same packed layer: %s" % PREFILL_OF[args.workload])
        extra["prefill"] = measure_prefill(layer, inputs, PREFILL_OF[args.workload], hip,
                                           args.prefill_steps, 5, bf16=not args.no_bf16)
        log("prefill", extra["prefill"])
    if not args.no_bf16 and not wk.redraw_every:
        # the unquantized 16-bit layer through the library's own kernels
        u = {"decode": measure_unquantized(args.workload, hip, min(K, 50), 5, ms_per_step)}
        if not args.no_prefill and args.workload in PREFILL_OF:
            u["prefill"] = measure_unquantized(PREFILL_OF[args.workload], hip, args.prefill_steps, 3,
                                               extra["prefill"]["ms_per_step"])
        extra["unquantized_16bit"] = u
        log("unquantized 16-bit", u)
    if not wk.redraw_every and not args.no_dataset_switch:
        # last: it rewrites the layer's copies
        extra["dataset_switch"] = measure_dataset_switch(layer, inputs, hip, ms_per_step)
        log("dataset switch", extra["dataset_switch"])

    if args.workload == "mixtral-decode" and not args.no_configs:
        # the other workloads, each on its own layer
        import moe_inputs as mi
        n = max(1, args.config_rotate)
        log("deepseek-decode / -prefill: packing %d copies" % n)
        ds = pack_copies(mi.WORKLOADS["deepseek-decode"], n)
        extra["deepseek_decode"] = measure_decode_config("deepseek-decode", ds, hip, min(K, 100), 5)
        log("deepseek decode", extra["deepseek_decode"])
        extra["deepseek_prefill"] = measure_prefill(ds[0][0], ds[0][1], "deepseek-prefill", hip,
                                                    args.prefill_steps, 5, bf16=False)
        log("deepseek prefill", extra["deepseek_prefill"])
        ds.clear()
        torch.cuda.empty_cache()
        if not args.no_bf16:
            extra["deepseek_unquantized_16bit"] = {
                # against the cache-defeated (rotated) quantized step: the 16-bit layer
                # (1.1 GB) does not fit the Infinity Cache either
                "decode": measure_unquantized("deepseek-decode", hip, min(K, 50), 5,
                                              extra["deepseek_decode"]["ms_per_step"]),
                "prefill": measure_unquantized("deepseek-prefill", hip, args.prefill_steps, 3,
                                               extra["deepseek_prefill"]["ms_per_step"])}
            log("deepseek unquantized 16-bit", extra["deepseek_unquantized_16bit"])
        log("qwen-stress: %d copies, %d steps" % (n, mi.WORKLOADS["qwen-stress"].steps))
        extra["qwen_stress"] = measure_stress(hip, n)
        log("qwen stress", extra["qwen_stress"])

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle for at least %.0f s ..." % args.cpu_seconds)
        cpu = cpu_baseline(wk, inputs, batch, args.cpu_seconds)
        log("cpu baseline", cpu)

    # The binding roof of the gate/up launch: its algorithmic bytes at HBM
    # peak against its algorithmic flops at the bf16 MFMA peak.
    hbm_bound = byt["gate_up"] / HBM_PEAK_GBS >= flops_gate_up(layer, offsets) / 1e3 / BF16_PEAK_TFLOPS
    kernel = ("FFN gate/up stage (gate+up projections, SiLU-GLU epilogue): ffn_stream_kernel "
              "for up to 28 tokens per expert (48 for experts narrower than d_ff 4096; shared "
              "experts up to 512 tokens), else tile_plan_kernel + ffn_tile_kernel; routed and "
              "shared experts in one launch per kernel")
    if hbm_bound:
        roof = {"bound": "hbm", "kernel": kernel, "achieved": round(achieved_gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(args.workload),
                "algorithmic_bytes_per_launch": int(byt["gate_up"]),
                "avg_launch_ms": round(gu_ms, 5)}
    else:
        roof = {"bound": "mfma", "kernel": kernel, "achieved": round(achieved_tf, 2),
                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved_tf / BF16_PEAK_TFLOPS, 4),
                "traffic": measured_traffic(args.workload),
                "algorithmic_flops_per_launch": int(flops_gate_up(layer, offsets)),
                "avg_launch_ms": round(gu_ms, 5)}
    out = {
        "metric": "MoE-layer tokens/sec at decode & prefill; HBM GB/s / MFMA util vs peak",
        "value": round(tokens_per_s, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) bf16 activations with outlier "
                "columns)",
        "config": describe(wk),
        "roofline": roof,
        "cpu_baseline": cpu,
        **extra,
        "detail": {
            "host_enqueue_ms_per_step": round(enqueue / K * 1e3, 5),
            "diagnostic_step_ms": round(float(layer_ms.mean()), 5),
            "diagnostic_step_ms_p10_p50_p90": [round(float(np.percentile(layer_ms, q)), 5)
                                               for q in (10, 50, 90)],
            "stage_ms": {"xsum": round(float(st[0]), 5), "gate_up": round(float(st[1]), 5),
                         "hsum": round(float(st[2]), 5), "down": round(float(st[3]), 5)},
            "ffn_ms": round(ffn_ms, 5),
            "ffn_weight_bytes": int(byt["gate_up"] + byt["down"]),
            "ffn_gbs": round(ffn_gbs, 1), "ffn_hbm_frac": round(ffn_gbs / HBM_PEAK_GBS, 4),
            "ffn_tflops": round(flops / (ffn_ms * 1e-3) / 1e12, 3),
            "ffn_mfma_frac": round(flops / (ffn_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 5),
            "wall_ms_per_step": round(wall / K * 1e3, 5),
            "expert_rows": [int(v) for v in np.diff(offsets)],
        },
    }
    print(json.dumps(out), flush=True)
    reap_children()


if __name__ == "__main__":
    main()
