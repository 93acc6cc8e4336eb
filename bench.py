"""Decode-attention benchmark over a per-layer compressed KV cache on one MI355X.

Workload (default): the Qwen2.5-14B-shaped mixed stack — 48 layers, 40 query /
8 KV heads, head dim 128, batch 32, context 8192, a seeded plan with 16 layers
inheriting an earlier anchor's cache and anchor precisions drawn from
{bf16, int8, int4, int2} (KIVI32 grouped quantisation).  Synthetic seeded inputs
of that shape (keys with per-channel log-normal outliers).

A step is one decode step over all 48 layers: the split attention kernel (D1)
and the log-sum-exp merge (C1).  The cache is written once beforehand by the
prefill kernel (W1), which is timed separately and reported under
"prefill_write"; the decode-time append of one token to every layer (the tail
write, and every 32nd token the group write) is timed after the decode steps and
reported under "append".  `value` is algorithmic compressed-cache bytes read per step
(each distinct anchor once) divided by the step time, with everything resident
in HBM.  The CPU baseline is the oracle (test infrastructure) timed on a bounded
sample of the same workload.

With --config 3 the workload is the MLA-style stack instead (32 layers, 32 heads,
latent 512 + 64 kept to a per-layer width drawn from {512, 256, 128, 64}, batch 16,
context 16384; --variant int4 for a KIVI32 4-bit latent; --variant 14b / 14b-int4
for Qwen2.5-14B's latent shape: 48 layers, 40 heads, latent 1024 + 64, batch 32,
context 8192): a step is the absorbed query (A1), the latent decode (D2) and the
merge with the W_UV up-projection (C2).  The MLA line also times the prefill write
with the down-projection from hidden states of the model width.

Before its W warm-up steps the decode runs untimed for about 0.25 s (settle()):
after the prefill write, or an idle second, the GPU's clocks take tens of
milliseconds to settle (14B mixed stack: the first 14 steps after the write at
3360-3385 us, then 3260 us; after 1 s idle 3650 us falling to 3260 within 8
steps), so that W warm-ups alone would time part of that ramp instead of the
steady decode.  Every timed step still does the whole step's work.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attention cache GB/s (% of HBM peak) and µs/step, 14B-shaped b=32 ctx=8k"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16/bf16 matrix peak


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--variant", default=None)
    ap.add_argument("--qscheme", default="kivi32", choices=["kivi32", "symrow", "group64"],
                    help="quantiser of the quantised layers (group64: GQA workloads only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--per-sequence", action="store_true",
                    help="workloads 2 and 3 with a plan per sequence (each drawn like the shared one)")
    ap.add_argument("--cpu-layers", type=int, default=0, help="layers in the CPU sample (0: auto)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of known size (counter calibration)")
    ap.add_argument("--selector-tokens", type=int, default=0,
                    help="only time the selector forward pass at this many prompt tokens "
                         "(workload 2's embedding width and layers)")
    return ap.parse_args()


# Counter records (scaled FETCH_SIZE + WRITE_SIZE per launch of the roofline kernel),
# per workload, with the sources that determine that kernel and its launch shape.
GQA_SOURCES = ["table.cpp", "decode.hip", "kvk_device.h", "kvk_internal.h"]
MLA_SOURCES = ["table.cpp", "mla.hip", "kvk_device.h", "kvk_internal.h"]
QS_NAMES = {0: "KIVI32", 1: "SYMROW", 2: "GROUP64"}
TRAFFIC = {
    (2, None): ("gqa_decode_14b_mixed_traffic.json", GQA_SOURCES),
    (3, None): ("mla_decode_32l_bf16_traffic.json", MLA_SOURCES),
    (3, "int4"): ("mla_decode_32l_int4_traffic.json", MLA_SOURCES),
}


def time_append(kvk, torch, table, n_layers, arena, n_stored, k_shape, v_shape, dev):
    """Decode-time append of one token to every layer (one kvk_append_token call per
    token), timed over the last 32-token group of the streams: positions
    n_stored - 32 .. n_stored - 1, 31 tail writes then the write that completes the
    group and quantises it into the last full block.  Runs after the decode timing
    (it rewrites that block with new tokens)."""
    if n_stored < 32:
        return None
    g = torch.Generator(device=dev)
    g.manual_seed(77)
    kn = torch.randn(k_shape, generator=g, device=dev).to(torch.bfloat16)
    vn = torch.randn(v_shape, generator=g, device=dev).to(torch.bfloat16)
    p0 = n_stored - 32
    kvk.append_token(table, 0, n_layers, kn, vn, p0, arena)  # warm-up (a tail write)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(32)]
    torch.cuda.synchronize()
    for i in range(32):
        ev[i][0].record()
        kvk.append_token(table, 0, n_layers, kn, vn, p0 + i, arena)
        ev[i][1].record()
    torch.cuda.synchronize()
    us = [a.elapsed_time(b) * 1e3 for a, b in ev]
    return {"layers": n_layers, "us_tail_write": round(sum(us[:31]) / 31, 2), "us_group_write": round(us[31], 2),
            "us_per_token": round(sum(us) / 32, 2)}


def time_selector(kvk, torch, d_model, n_layers, dev, lengths=(2048, 8192, 32768)):
    """The selector forward pass (prompt embeddings -> plan) at several prompt lengths,
    synthetic weights of the model's embedding width, the GQA action space (depth and
    precision: 5 actions): µs per prompt, 4 warm-ups then the median of 12 (the
    paper's timing protocol)."""
    import numpy as np
    g = torch.Generator(device=dev)
    g.manual_seed(99)
    n_w = kvk.selector_weight_elems(d_model, n_layers, kvk.SELECTOR_ACTIONS_GQA)
    weights = (torch.randn(n_w, generator=g, device=dev) * 0.02).to(torch.bfloat16)
    actions = torch.empty(n_layers, dtype=torch.int32, device=dev)
    out = {}
    for T in lengths:
        emb = torch.randn((T, d_model), generator=g, device=dev).to(torch.bfloat16)
        ws = torch.empty(kvk.selector_workspace_bytes(d_model, n_layers, T), dtype=torch.uint8, device=dev)
        for _ in range(4):
            kvk.selector_forward(d_model, n_layers, weights, emb, actions, ws)
        times = []
        for _ in range(12):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            kvk.selector_forward(d_model, n_layers, weights, emb, actions, ws)
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e3)
        out[str(T)] = round(float(np.median(times)), 1)
        del emb, ws
    return {"d_model": d_model, "layers": n_layers, "actions": kvk.SELECTOR_ACTIONS_GQA,
            "us_by_prompt_tokens": out}


def kernel_source_hash(sources=GQA_SOURCES) -> str:
    """sha256 over the sources that determine a decode kernel and its splits."""
    import hashlib
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, "paper_2609_37988_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(config: int, variant=None, qscheme="kivi32"):
    """HBM bytes per launch of the roofline kernel from the committed counter record,
    or None when there is no record for this workload and quantiser (the records are
    KIVI32's) or it was taken on different kernel sources."""
    if qscheme != "kivi32" or (config, variant) not in TRAFFIC:
        return None
    name, sources = TRAFFIC[(config, variant)]
    try:
        with open(os.path.join(ROOT, "profiles", name)) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_hash(sources) or rec.get("config") != config:
        return None
    return rec.get("traffic_bytes_per_launch")


def calibrate_copy():
    """A plain device-to-device copy of 4 GiB, three times: the reference that scales
    the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    n = 4 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copies": 3}), flush=True)


def hbm_context(torch, dev, n=4 << 30):
    """Context for the roofline, not a target: the rates of torch's own device copy
    (reads and writes n bytes) and of a sum over n bytes (reads them), the median of
    10 after 3 warm-ups, on the same GPU in the same process."""
    src = torch.empty(n // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return sorted(ts)[len(ts) // 2]

    t_copy = timed(lambda: dst.copy_(src))
    t_sum = timed(lambda: src.sum())
    del src, dst
    torch.cuda.empty_cache()
    return {"copy_GB_per_s": round(2 * n / t_copy / 1e9, 1), "sum_read_GB_per_s": round(n / t_sum / 1e9, 1),
            "bytes": n, "kernels": "torch copy_ and sum, not this library's"}


def settle(torch, step, ms=250.0, max_steps=400):
    """Run step(i) untimed until about `ms` of wall time has passed (synchronising
    every 8 steps) so that the GPU's clocks have settled before the warm-up steps."""
    t0 = time.perf_counter()
    i = 0
    while i < max_steps:
        step(i)
        i += 1
        if i % 8 == 0:
            torch.cuda.synchronize()
            if (time.perf_counter() - t0) * 1e3 >= ms:
                break
    torch.cuda.synchronize()
    return i


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def median_of_12(torch, step):
    """App. B's timing protocol: four warm-ups, then twelve steps each between device
    synchronisations; the median in µs (reported beside the contract's mean)."""
    import numpy as np
    for i in range(4):
        step(i)
    times = []
    for i in range(12):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        step(i)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3)
    return round(float(np.median(times)), 1)


def host_cpu():
    """The host the CPU baseline runs on: CPU model (/proc/cpuinfo), logical CPUs
    (nproc) and the CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def cpu_baseline(w, table, n_stored, scale, n_layers_sample, n_batch=1):
    """Time the oracle's decode (dequantise + fp64 attention) for the first n_batch
    batch elements over the first n_layers_sample layers; inputs drawn on the CPU
    with the same recipe and compressed by the oracle beforehand (untimed)."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from oracle import attention as OA
    from oracle import cache as OC
    from oracle import plan as OP
    from paper_2609_37988_amd import kvk, synth

    d = table.dims
    od = OP.Dims(OP.GQA, d.n_layers, d.n_q_heads, d.n_kv_heads, d.head_dim, qscheme=d.qscheme,
                 batch=1, max_tokens=d.max_tokens, keep_tokens=d.keep_tokens)
    info = kvk.table_query(table)
    anc = info.anchor_of[:n_layers_sample]
    G = d.n_q_heads // d.n_kv_heads
    streams = {}
    for a in sorted(set(anc)):
        k, v = synth.kv_layer(w, a, device="cpu", batch=n_batch)
        keep = None
        if w.keep_tokens:
            keep = synth.keep_positions(w, a, device="cpu", batch=n_batch).numpy()
        kn, vn = k.float().numpy(), v.float().numpy()
        bits = w.plan[a][1]
        for b in range(n_batch):
            for h in range(d.n_kv_heads):
                kk, vv = kn[b, h], vn[b, h]
                if keep is not None:
                    kk, vv = OC.gather_kept(kk, keep[b, h]), OC.gather_kept(vv, keep[b, h])
                streams[(a, b, h)] = (bits, OC.compress_stream(od, bits, kk, vv))
    q = synth.queries(w, n_layers_sample, device="cpu", batch=n_batch).float().numpy().astype(np.float64)
    t0 = time.perf_counter()
    for b in range(n_batch):
        for l in range(n_layers_sample):
            for h in range(d.n_kv_heads):
                bits, st = streams[(anc[l], b, h)]
                K, V = OC.dequant_stream(od, bits, st, n_stored)
                OA.softmax_attention(q[l, b, h * G:(h + 1) * G], K, V, scale)
    dt = time.perf_counter() - t0
    sample_bytes = kvk.read_bytes(table, 0, n_layers_sample, n_stored) // d.batch * n_batch
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(sample_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"batch elements 0..{n_batch - 1} of {d.batch}, layers 0..{n_layers_sample - 1} "
                      f"({len(set(anc))} anchors x {d.n_kv_heads} KV heads), {n_stored} tokens: "
                      f"{sample_bytes} algorithmic bytes in {dt:.2f} s (numpy fp64 oracle; "
                      f"elementwise work single-threaded, BLAS threads = cores)",
            "seconds": round(dt, 3), **host_cpu()}


def cpu_baseline_mla(w, table, n_stored, scale, n_layers_sample):
    """Time the oracle's MLA decode (dequantise, reconstruct keys and values with the
    up-projections, fp64 attention) for batch element 0 over the first
    n_layers_sample layers; inputs compressed by the oracle beforehand (untimed)."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import mla as OM
    from oracle import plan as OP
    from paper_2609_37988_amd import kvk, synth

    d = table.dims
    od = OP.Dims(OP.MLA, d.n_layers, d.n_q_heads, d.n_kv_heads, d.head_dim, latent_dim=d.latent_dim,
                 rope_dim=d.rope_dim, nope_dim=d.nope_dim, v_dim=d.v_dim, qscheme=d.qscheme, batch=1,
                 max_tokens=d.max_tokens, keep_tokens=d.keep_tokens)
    info = kvk.table_query(table)
    anc = info.anchor_of[:n_layers_sample]
    streams = {}
    for a in sorted(set(anc)):
        c, r = synth.mla_layer(w, a, device="cpu", batch=1)
        _, bits, rank = w.plan[a]
        streams[a] = (bits, rank, OM.compress_stream(od, bits, rank, c[0].float().numpy(), r[0].float().numpy()))
    q = synth.mla_queries(w, n_layers_sample, device="cpu", batch=1).float().numpy().astype(np.float64)
    wk, wv = synth.mla_weights(w, n_layers_sample, device="cpu")
    wk, wv = wk.float().numpy().astype(np.float64), wv.float().numpy().astype(np.float64)
    nope = d.nope_dim
    t0 = time.perf_counter()
    for l in range(n_layers_sample):
        bits, rank, st = streams[anc[l]]
        C, R = OM.dequant_stream(od, bits, rank, st, n_stored)
        OM.attention_reconstructed(q[l, 0, :, :nope], q[l, 0, :, nope:], C, R, wk[l], wv[l], scale)
    dt = time.perf_counter() - t0
    sample_bytes = kvk.read_bytes(table, 0, n_layers_sample, n_stored) // d.batch
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"value": round(sample_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"batch element 0 of {d.batch}, layers 0..{n_layers_sample - 1} "
                      f"({len(set(anc))} anchors), {n_stored} tokens: {sample_bytes} algorithmic bytes "
                      f"in {dt:.2f} s (numpy fp64 oracle, keys and values reconstructed with the "
                      f"up-projections; BLAS threads = cores)",
            "seconds": round(dt, 3), **host_cpu()}


def run_mla(args):
    """The MLA-style stack: prefill write (W2), then timed decode steps (A1 + D2, C2)."""
    import numpy as np
    import torch

    from paper_2609_37988_amd import kvk, synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.mla_workload(args.variant)
    if args.qscheme == "group64":
        print("bench.py: the GROUP64 quantiser is built for GQA tables only", file=sys.stderr)
        sys.exit(2)
    if args.qscheme == "symrow":
        w.qscheme = kvk.SYMROW
    n_tok = w.tokens
    n_stored = w.keep_tokens if w.keep_tokens else n_tok
    dims = kvk.make_dims(kvk.MLA, w.n_layers, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, w.latent_dim,
                         w.rope_dim, w.nope_dim, w.v_dim, qscheme=w.qscheme, batch=w.batch,
                         max_tokens=n_tok, keep_tokens=w.keep_tokens)
    plans = None
    if args.per_sequence:  # each sequence its own kept widths (drawn like the shared plan)
        plans = synth.mla_plans_per_sequence(w)
        table = kvk.layer_table_batched(dims, [kvk.make_plan(p) for p in plans])
        w.name += "-per-sequence"
    else:
        table = kvk.layer_table(dims, kvk.make_plan(w.plan))
    info = kvk.table_query(table)
    log(f"workload {w.name}: arena {info.arena_bytes / 1e9:.2f} GB, rho eq.(2) {info.rho:.2f}, "
        f"anchors {info.n_anchors}")
    arena = torch.empty(info.arena_bytes, dtype=torch.uint8, device=dev)
    w2_ms, w2_bytes = 0.0, 0
    for l in range(w.n_layers):
        if w.plan[l][0]:
            continue
        c, r = synth.mla_layer(w, l, device=dev)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        kvk.compress_layer(table, l, c, r, n_tok, None, arena)
        e1.record()
        torch.cuda.synchronize()
        w2_ms += e0.elapsed_time(e1)
        if plans is None:
            w2_bytes += w.batch * n_tok * (w.plan[l][2] + w.rope_dim) * c.element_size() + info.layer_bytes[l]
        else:
            for b, p in enumerate(plans):
                if not p[l][0]:
                    w2_bytes += n_tok * (p[l][2] + w.rope_dim) * c.element_size() + \
                        kvk.table_sequence_query(table, b).layer_bytes[l]
        del c, r
    torch.cuda.empty_cache()
    log(f"prefill write: {w2_ms:.1f} ms over {info.n_anchors} anchors")

    qs = [synth.mla_queries(w, w.n_layers, device=dev) for _ in range(1)]
    qs.append(qs[0].flip(1).contiguous())  # a second query set: sequences reversed
    wk, wv = synth.mla_weights(w, w.n_layers, device=dev)
    wk = kvk.mla_weights_for_library(wk)  # arranged once, as at weight load
    out = torch.empty((w.n_layers, w.batch, w.n_q_heads, w.v_dim), dtype=torch.float32, device=dev)
    ws = torch.empty(kvk.workspace_bytes(table, 0, w.n_layers), dtype=torch.uint8, device=dev)
    kvk.decode_setup(table, 0, w.n_layers, ws)  # per-sequence plans: the work list, once
    scale = w.softmax_scale()
    alg = kvk.read_bytes(table, 0, w.n_layers, n_stored)
    settle(torch, lambda i: kvk.decode_attention(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, out, ws,
                                                 w_uk=wk, w_uv=wv))
    for i in range(args.warmup):
        kvk.decode_attention(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, out, ws, w_uk=wk, w_uv=wv)
    torch.cuda.synchronize()
    K = args.steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for i in range(K):
        ev[i][0].record()
        kvk.decode_splits(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, ws, w_uk=wk, w_uv=wv)
        ev[i][1].record()
        kvk.decode_merge(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, ws, out, w_uk=wk, w_uv=wv)
    t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / K
    sp_avg = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    gbs = alg / (ms_step * 1e-3) / 1e9
    sp_gbs = alg / (sp_avg * 1e-3) / 1e9
    med12 = median_of_12(torch, lambda i: kvk.decode_attention(table, 0, w.n_layers, qs[i % 2], n_stored, scale,
                                                               arena, out, ws, w_uk=wk, w_uv=wv))
    # the kept width each (sequence, layer) reads: its plan's anchor's
    seq_plans = plans if plans is not None else [w.plan] * w.batch
    seq_infos = [kvk.table_sequence_query(table, b) for b in range(w.batch)] if plans is not None else [info] * w.batch
    kept = [[p[si.anchor_of[l]][2] for l in range(w.n_layers)] for p, si in zip(seq_plans, seq_infos)]
    # up-projection bytes: once per layer with one plan, once per sequence and layer with one per sequence
    wbytes = sum(w.n_q_heads * (w.nope_dim + w.v_dim) * d * 2
                 for kb in (kept if plans is not None else kept[:1]) for d in kb)
    # matrix-core work of D2 per step: scores over the W = d + d_R stored channels and
    # the probability-by-latent product over d, per (token, head), 2 flops per MAC
    d2_flops = sum(2 * n_stored * w.n_q_heads * (2 * d + w.rope_dim) for kb in kept for d in kb)
    log(f"step {ms_step * 1e3:.1f} us, {gbs:.1f} GB/s ({100 * gbs / HBM_PEAK_GBS:.1f}% of HBM); "
        f"A1+D2 {sp_avg * 1e3:.1f} us ({sp_gbs:.1f} GB/s)")
    app = time_append(kvk, torch, table, w.n_layers, arena, n_stored, (w.n_layers, w.batch, w.latent_dim),
                      (w.n_layers, w.batch, w.rope_dim), dev)
    log(f"append: {app}")
    proj = time_projected_write(kvk, torch, w, table, arena, n_tok, dev, plans)
    log(f"projected write: {proj}")
    snap = time_snapkv_mla(kvk, torch, w, dev) if plans is None else None
    log(f"snapkv (MLA): {snap}")
    ctx = hbm_context(torch, dev)
    log(f"HBM context: {ctx}")
    cpu = None  # last: its host thread pool would delay the launch-bound timings above
    if not args.no_cpu_baseline and plans is None:
        cpu = cpu_baseline_mla(w, table, n_stored, scale, min(args.cpu_layers or 32, w.n_layers))
        log(f"cpu baseline: {cpu['value']} GB/s over {cpu['seconds']} s")
    ranks = {}
    for p in (seq_plans if plans is not None else [w.plan]):
        for e in p:
            if not e[0]:
                ranks[str(e[2])] = ranks.get(str(e[2]), 0) + 1
    line = {
        "metric": METRIC, "value": round(gbs, 2), "unit": "GB/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "us_per_step": round(ms_step * 1e3, 2),
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("bf16" if w.plan[0][1] == 16 else f"u{w.plan[0][1]}") + " latent cache; f16/bf16 MFMA, f32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": w.name, "layers": w.n_layers, "q_heads": w.n_q_heads, "latent_dim": w.latent_dim,
            "rope_dim": w.rope_dim, "batch": w.batch, "context": n_tok, "stored_tokens": n_stored,
            "qscheme": QS_NAMES[w.qscheme], "anchors_by_rank": ranks,
            "bits": w.plan[0][1], "rho_eq2": round(info.rho, 3), "alg_bytes_per_step": alg,
            "up_projection_bytes_per_step": wbytes,
        },
        "roofline": {
            "bound": "hbm", "kernel": "mla_absorb_kernel + mla_decode_kernel (A1 + D2)",
            "achieved": round(sp_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(sp_gbs / HBM_PEAK_GBS, 4),
            "traffic": recorded_traffic(3, args.variant) if args.qscheme == "kivi32" else None,
            "launch_us": round(sp_avg * 1e3, 2), "bytes_per_launch": alg,
        },
        "mfma": {"flops_per_step": d2_flops, "achieved": round(d2_flops / (sp_avg * 1e-3) / 1e12, 1),
                 "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                 "frac": round(d2_flops / (sp_avg * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 4)},
        "cpu_baseline": cpu,
        "hbm_context": ctx,
        "prefill_write": {"ms": round(w2_ms, 3), "bytes": w2_bytes,
                          "GB_per_s": round(w2_bytes / (w2_ms * 1e-3) / 1e9, 2)},
        "median_of_12_us_per_step": med12,
        "append": app,
        "prefill_write_projected": proj,
        "snapkv_select_mla": snap,
    }
    print(json.dumps(line), flush=True)


def time_projected_write(kvk, torch, w, table, arena, n_tok, dev, plans=None):
    """The prefill write with the down-projection (kvk_compress_layer_project) of the
    widest anchor, from hidden states of the model width: median of 5 after 2 warmups.
    With one plan per sequence: layer 0, which every plan stores, each sequence at its
    own kept width.  Runs after the decode timing (it rewrites that layer's region)."""
    from paper_2609_37988_amd import synth
    if plans is None:
        anchors = [l for l in range(w.n_layers) if not w.plan[l][0]]
        l = max(anchors, key=lambda a: w.plan[a][2])
        d, bits = w.plan[l][2], w.plan[l][1]
        widths = [d] * w.batch
    else:
        l = 0
        widths = [p[l][2] for p in plans]
        d, bits = sorted(set(widths)), sorted({p[l][1] for p in plans})
    x = synth.latent_random(91, w.batch, n_tok, w.d_model, device=dev)
    wd = synth.weights_random(92, 1, 1, w.latent_dim, w.d_model, device=dev)[0, 0].contiguous()
    r = synth.latent_random(93, w.batch, n_tok, w.rope_dim, device=dev)
    for _ in range(2):
        kvk.compress_layer_project(table, l, x, wd, r, n_tok, None, arena)
    torch.cuda.synchronize()
    ts = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        kvk.compress_layer_project(table, l, x, wd, r, n_tok, None, arena)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = sorted(ts)[2]
    flops = 2.0 * n_tok * w.d_model * sum(widths)
    del x, wd, r
    torch.cuda.empty_cache()
    return {"layer": l, "d": d, "bits": bits, "d_model": w.d_model, "tokens": w.batch * n_tok,
            "us": round(ms * 1e3, 1), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
            "mfma_frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 4),
            "x_read_GB_per_s": round(w.batch * n_tok * w.d_model * 2 / (ms * 1e-3) / 1e9, 1)}


def time_snapkv_mla(kvk, torch, w, dev):
    """The query-aware keep list of one MLA anchor (kvk_snapkv_select_mla) at the
    stack's shape, keeping half of the positions: median of 5 after 2 warmups.  Bytes:
    the latent and positional keys read by both score passes; matrix-core work: the
    window rows' scores (32 queries x every head) against the full-width latent, twice."""
    from paper_2609_37988_amd import synth
    n = w.tokens
    dims = kvk.make_dims(kvk.MLA, 1, w.n_q_heads, w.ref_kv_heads, w.ref_head_dim, w.latent_dim, w.rope_dim,
                         w.nope_dim, w.v_dim, qscheme=w.qscheme, batch=w.batch, max_tokens=n, keep_tokens=n // 2)
    t = kvk.layer_table(dims, kvk.make_plan([(0, 16, w.latent_dim)]))
    c = synth.latent_random(95, w.batch, n, w.latent_dim, device=dev)
    r = synth.latent_random(96, w.batch, n, w.rope_dim, device=dev)
    q = synth.q_random(97, w.batch, 32, w.n_q_heads, w.nope_dim + w.rope_dim, device=dev)
    wk = kvk.mla_weights_for_library(synth.weights_random(98, 1, w.n_q_heads, w.nope_dim, w.latent_dim,
                                                          device=dev))[0]
    keep = torch.empty((w.batch, n // 2), dtype=torch.int32, device=dev)
    ws = torch.empty(kvk.snapkv_workspace_bytes(t, n), dtype=torch.uint8, device=dev)
    scale = w.softmax_scale()
    for _ in range(2):
        kvk.snapkv_select_mla(t, 0, c, r, q, n, scale, keep, ws, w_uk=wk)
    torch.cuda.synchronize()
    ts = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        kvk.snapkv_select_mla(t, 0, c, r, q, n, scale, keep, ws, w_uk=wk)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = sorted(ts)[2]
    width = w.latent_dim + w.rope_dim
    nbytes = 2 * w.batch * n * width * 2
    flops = 2 * 2.0 * w.batch * n * 32 * w.n_q_heads * width
    del c, r, q, wk, ws
    torch.cuda.empty_cache()
    return {"batch": w.batch, "tokens": n, "keep": n // 2, "q_heads": w.n_q_heads, "latent_dim": w.latent_dim,
            "us": round(ms * 1e3, 1), "key_reads_GB_per_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1)}


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for {args.gpus} GPUs).", file=sys.stderr)
        sys.exit(2)
    if args.config == 3:
        run_mla(args)
        return
    if args.selector_tokens > 0:
        import torch

        from paper_2609_37988_amd import kvk, synth

        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        w = synth.workload(2)
        sel = time_selector(kvk, torch, w.n_q_heads * w.head_dim, w.n_layers, dev, lengths=(args.selector_tokens,))
        print(json.dumps({"selector_forward": sel}), flush=True)
        return
    import numpy as np
    import torch

    from paper_2609_37988_amd import kvk, synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.workload(args.config, args.variant)
    if args.qscheme == "symrow":
        w.qscheme = kvk.SYMROW
    elif args.qscheme == "group64":
        w.qscheme = kvk.GROUP64
    n_tok = w.tokens
    n_stored = w.keep_tokens if w.keep_tokens else n_tok
    dims = kvk.make_dims(kvk.GQA, w.n_layers, w.n_q_heads, w.n_kv_heads, w.head_dim, qscheme=w.qscheme,
                         batch=w.batch, max_tokens=n_tok, keep_tokens=w.keep_tokens)
    plans = None
    if args.per_sequence:
        if args.config != 2:
            print("--per-sequence applies to workload 2", file=sys.stderr)
            sys.exit(2)
        plans = synth.plans_per_sequence(w)
        table = kvk.layer_table_batched(dims, [kvk.make_plan(p) for p in plans])
    else:
        table = kvk.layer_table(dims, kvk.make_plan(w.plan))
    info = kvk.table_query(table)
    log(f"workload {w.name}: arena {info.arena_bytes / 1e9:.2f} GB, rho eq.(2) {info.rho:.2f}, "
        f"realized {info.rho_realized:.2f}, anchors {info.n_anchors}")
    arena = torch.empty(info.arena_bytes, dtype=torch.uint8, device=dev)

    # ---- prefill write (W1), timed per anchor layer ----
    # With eviction, the query-aware keep list (kvk_snapkv_select) is also timed on
    # each anchor's keys; the cache keeps the workload's seeded subset.
    w1_ms, w1_bytes = 0.0, 0
    snap_ms, snap_bytes, snap_flops = 0.0, 0, 0
    if w.keep_tokens:
        snap_ws = torch.empty(kvk.snapkv_workspace_bytes(table, n_tok), dtype=torch.uint8, device=dev)
        snap_keep = torch.empty((w.batch, w.n_kv_heads, w.keep_tokens), dtype=torch.int32, device=dev)
        q_obs = synth.q_random(4242, w.batch, w.n_q_heads, 32, w.head_dim, device=dev)
    for l in range(w.n_layers):
        if (w.plan[l][0] if plans is None else all(p[l][0] for p in plans)):
            continue
        k, v = synth.kv_layer(w, l, device=dev)
        keep = synth.keep_positions(w, l, device=dev) if w.keep_tokens else None
        if w.keep_tokens:
            kvk.snapkv_select(table, l, k, q_obs, n_tok, w.softmax_scale(), snap_keep, snap_ws)  # warm
            torch.cuda.synchronize()
            s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s0.record()
            kvk.snapkv_select(table, l, k, q_obs, n_tok, w.softmax_scale(), snap_keep, snap_ws)
            s1.record()
            torch.cuda.synchronize()
            snap_ms += s0.elapsed_time(s1)
            snap_bytes += 2 * k.numel() * k.element_size() + q_obs.numel() * q_obs.element_size()
            snap_flops += 2 * 2 * w.batch * w.n_q_heads * 32 * n_tok * w.head_dim
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        kvk.compress_layer(table, l, k, v, n_tok, keep, arena)
        e1.record()
        torch.cuda.synchronize()
        w1_ms += e0.elapsed_time(e1)
        if plans is None:
            w1_bytes += 2 * k.numel() * k.element_size() * n_stored // n_tok + info.layer_bytes[l]
        else:
            for b, p in enumerate(plans):
                if not p[l][0]:
                    w1_bytes += (2 * k[b].numel() * k.element_size() * n_stored // n_tok +
                                 kvk.table_sequence_query(table, b).layer_bytes[l])
        del k, v, keep
    torch.cuda.empty_cache()
    log(f"prefill write: {w1_ms:.1f} ms over {info.n_anchors} anchors")

    qs = [synth.queries(w, w.n_layers, device=dev, seed_offset=i) for i in range(2)]
    out = torch.empty((w.n_layers, w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device=dev)
    ws = torch.empty(kvk.workspace_bytes(table, 0, w.n_layers), dtype=torch.uint8, device=dev)
    kvk.decode_setup(table, 0, w.n_layers, ws)  # per-sequence plans: the work list, once
    scale = w.softmax_scale()
    alg = kvk.read_bytes(table, 0, w.n_layers, n_stored)

    settle(torch, lambda i: kvk.decode_attention(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, out, ws))
    for i in range(args.warmup):
        kvk.decode_attention(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, out, ws)
    torch.cuda.synchronize()
    K = args.steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for i in range(K):
        ev[i][0].record()
        kvk.decode_splits(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, ws)
        ev[i][1].record()
        kvk.decode_merge(table, 0, w.n_layers, qs[i % 2], n_stored, scale, arena, ws, out)
    t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / K
    d1_ms = [a.elapsed_time(b) for a, b in ev]
    d1_avg = float(np.mean(d1_ms))
    gbs = alg / (ms_step * 1e-3) / 1e9
    d1_gbs = alg / (d1_avg * 1e-3) / 1e9
    log(f"step {ms_step * 1e3:.1f} us, {gbs:.1f} GB/s ({100 * gbs / HBM_PEAK_GBS:.1f}% of HBM); "
        f"D1 {d1_avg * 1e3:.1f} us ({d1_gbs:.1f} GB/s)")
    med12 = median_of_12(torch, lambda i: kvk.decode_attention(table, 0, w.n_layers, qs[i % 2], n_stored, scale,
                                                               arena, out, ws))
    log(f"paper's protocol (4 warm-ups, median of 12 synchronised steps): {med12} us")

    app = time_append(kvk, torch, table, w.n_layers, arena, n_stored,
                      (w.n_layers, w.batch, w.n_kv_heads, w.head_dim), (w.n_layers, w.batch, w.n_kv_heads, w.head_dim),
                      dev)
    log(f"append: {app}")
    sel = time_selector(kvk, torch, w.n_q_heads * w.head_dim, w.n_layers, dev) if args.config == 2 else None
    log(f"selector: {sel}")
    ctx = hbm_context(torch, dev)
    log(f"HBM context: {ctx}")
    # The CPU baseline runs last: its host thread pool, busy for seconds, would
    # otherwise delay the launches of the launch-bound timings above.
    cpu = None
    if not args.no_cpu_baseline and plans is None:
        nl = args.cpu_layers or (w.n_layers if args.config in (1, 2) else 4)
        cpu = cpu_baseline(w, table, n_stored, scale, nl, n_batch=2 if args.config in (1, 2) else 1)
        log(f"cpu baseline: {cpu['value']} GB/s over {cpu['seconds']} s")

    bits_mix = {}
    for p in ([w.plan] if plans is None else plans):
        for e in p:
            if not e[0]:
                bits_mix[str(e[1])] = bits_mix.get(str(e[1]), 0) + 1
    line = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "us_per_step": round(ms_step * 1e3, 2),
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u2/u4/u8 codes + bf16 cache; f16/bf16 MFMA, f32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": w.name + ("-per-sequence-plans" if plans else ""), "layers": w.n_layers,
            "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads,
            "head_dim": w.head_dim, "batch": w.batch, "context": n_tok, "stored_tokens": n_stored,
            "qscheme": QS_NAMES[w.qscheme],
            "anchors_by_bits": bits_mix,
            "inheriting_layers": sum(e[0] for p in ([w.plan] if plans is None else plans) for e in p),
            "rho_eq2": round(info.rho, 3), "rho_realized": round(info.rho_realized, 3),
            "alg_bytes_per_step": alg,
        },
        "roofline": {
            "bound": "hbm", "kernel": "gqa_decode_kernel (D1)", "achieved": round(d1_gbs, 2),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(d1_gbs / HBM_PEAK_GBS, 4),
            "traffic": (recorded_traffic(args.config, args.variant)
                        if args.qscheme == "kivi32" and plans is None else None),
            "launch_us": round(d1_avg * 1e3, 2), "bytes_per_launch": alg,
        },
        "cpu_baseline": cpu,
        "prefill_write": {"ms": round(w1_ms, 3), "bytes": w1_bytes,
                          "GB_per_s": round(w1_bytes / (w1_ms * 1e-3) / 1e9, 2)},
        "append": app,
        "selector_forward": sel,
        "median_of_12_us_per_step": med12,
        "hbm_context": ctx,
    }
    if w.keep_tokens:
        line["snapkv_select"] = {
            "ms": round(snap_ms, 3), "anchors": info.n_anchors, "bytes": snap_bytes,
            "GB_per_s": round(snap_bytes / (snap_ms * 1e-3) / 1e9, 2),
            "TFLOP_per_s": round(snap_flops / (snap_ms * 1e-3) / 1e12, 1)}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
