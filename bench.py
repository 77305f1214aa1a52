#!/usr/bin/env python3
"""Benchmark of the fused suffix restore on one MI355X.

One step = one ``pkv_restore`` of the whole workload (every layer, every
reused block) from a device-resident checkpoint into device-resident paged
caches.  Prints one JSON line.  The checkpoint itself is written on the GPU
by ``pkv_quantize_gather`` from the drawn old caches; that write is timed too
and reported under ``checkpoint_write``.

    python bench.py [--steps K] [--warmup W] [--workload llama8b_32l] [--int4 K8V4|K4V4]

Throughput is algorithmic bytes (payload and scales of reused blocks read,
restored rows written) per second; the roofline entry divides the same bytes
by the restore kernel's average duration from HIP events on its stream.
The oracle, timed on the host cores on a bounded sample of the same
workload, is reported beside it as ``cpu_baseline``.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import multiprocessing as mp
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "restored KV GB/s + % HBM peak; µs to restore 32K-token suffix (8B shape)"
HBM_PEAK_GBPS = 8000.0
PCIE_PEAK_GBPS = 64.0  # PCIe 5.0 x16, one direction, before protocol overhead
KERNEL_SRC = os.path.join(ROOT, "paper_2609_26219_amd", "csrc", "restore.hip")
GATHER_SRC = os.path.join(ROOT, "paper_2609_26219_amd", "csrc", "gather.hip")

WORKLOAD_TEXT = {
    "llama8b_32l": "Llama-3-8B-shaped suffix restore: 32 layers x 8 KV heads x head_dim 128, 32768-token suffix, "
                   "block 32, page 16, bf16 cache, tag mix 70% int4 / 20% int8 / 10% fp16, 15% repair blocks, "
                   "delta -1500",
    "llama8b_1l": "Llama-3-8B-shaped single layer: 8 KV heads x head_dim 128, 8192-token suffix, block 32, page 16, "
                  "fp16 cache, 70/20/10 tag mix, 10% repair",
    "llama70b": "Llama-70B-shaped: 80 layers x 8 KV heads x head_dim 128, 65536-token suffix, block 64, page 32, "
                "bf16 cache, 60/30/10 tag mix, 12% repair, delta +4096",
    "tiny": "tiny: 1 layer x 2 KV heads x head_dim 64, 512 tokens, block 16",
    "batched16": "batched resumes: 16 requests on the 32-layer 8B shape, suffixes of 4096-65536 tokens, "
                 "per-request delta in [-8192, 8192] and Dirichlet tag mixes, 5-20% repair, one 2^20-slot paged pool "
                 "with interleaved page ownership",
}
# Workloads whose old caches of all layers do not fit beside the pool and the
# checkpoint: their checkpoint is written layer by layer (not timed), and one
# buffer set is used.
LAYERWISE = {"batched16"}


KV_LAYOUT_TEXT = {
    "paired": "paired: one cache [L][pool_pages][2][P][H][D], a page's K slots then its V slots",
    "separate": "separate: k_cache and v_cache, each [L][pool_pages][P][H][D]",
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_hash(src: str = KERNEL_SRC) -> str:
    return hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]


def measured_traffic(workload: str, int4: str, layout: str, kernel: str = "restore_kernel", src: str = KERNEL_SRC):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_{int4.lower()}_{layout}_pmc.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"^traffic-json: (\{.*\})\s*$", open(path).read(), re.M)
    if not m:
        return None
    d = json.loads(m.group(1))
    if d.get("kernel_sha256_16") != kernel_hash(src):
        return None
    return d.get("traffic_bytes_per_launch")


# ---------------------------------------------------------------------------
# CPU baseline: the oracle, per layer, in worker processes
# ---------------------------------------------------------------------------

def _oracle_layer(args):
    """One layer of one request: the oracle writes its checkpoint from the
    drawn rows (timed separately), then restores it (timed)."""
    import dataclasses

    import numpy as np

    import oracle
    from oracle import quantize as oq

    case, ri, layer = args
    req = case.requests[ri]
    _, kb, vb = case.suffix_bits(ri, layer)
    t = time.perf_counter()
    pb, sb = oq.quantize_rows(case.shape, req, kb, vb)
    t_write = time.perf_counter() - t
    one = dataclasses.replace(req, payload_offset=0, scale_offset=0)
    s1 = dataclasses.replace(case.shape, num_layers=1)
    H, D = s1.num_kv_heads, s1.head_dim
    k_cache = np.zeros((s1.pool_pages * s1.page_size, H, D), np.uint16)
    v_cache = np.zeros_like(k_cache)
    scales = sb.reshape(-1)
    # The oracle's restore body, block by block, into the caches in place
    # (oracle.restore itself first copies both caches, which is not part of
    # the method and would dominate on a 2^20-slot pool).
    t = time.perf_counter()
    layout = oracle.block_layout(req.tags, s1.block_tokens, H, D)
    for b in oracle.reused_blocks(one):
        slots, k, v = oracle.restore_block(pb, scales, s1, one, 0, b, layout)
        k_cache[slots] = oracle.round_to_output(k, s1.out_dtype)
        v_cache[slots] = oracle.round_to_output(v, s1.out_dtype)
    return time.perf_counter() - t, t_write


def cpu_baseline(case, pool, workers: int, target_layers: int = 32):
    """Oracle throughput on the host cores over a bounded sample of layers,
    one layer per job on ``pool`` (``workers`` processes, forked before the
    benchmark touched the GPU)."""
    layers = list(range(min(case.shape.num_layers, max(target_layers, workers))))
    jobs = [(case, 0, l) for l in layers]
    per_layer = pool.map(_oracle_layer, jobs) if pool is not None else [_oracle_layer(j) for j in jobs]
    # Each process times its own layer; the pool runs `workers` layers at once.
    restore_cpu = sum(t for t, _ in per_layer)
    write_cpu = sum(t for _, t in per_layer)
    rounds = -(-len(layers) // workers)
    wall = restore_cpu / len(layers) * rounds
    # One layer in this process alone: the single-worker rate, free of the pool's memory contention.
    one_layer_s, _ = _oracle_layer((case, 0, 0))
    per_layer_bytes = case.algorithmic_bytes()["total"] / case.shape.num_layers
    sample_bytes = per_layer_bytes * len(layers)
    return {
        "value": round(sample_bytes / wall / 1e9, 4),
        "unit": "GB/s",
        "cores": workers,
        "kind": "oracle",
        "sample": f"{len(layers)} of {case.shape.num_layers} layers of the same workload (request 0), one process "
                  f"per layer, {workers} processes; restore cpu {restore_cpu:.1f} s over {rounds} round(s) of "
                  f"{workers} layers; checkpoint write (oracle quantize-and-gather) cpu {write_cpu:.1f} s, untimed "
                  f"in value",
        "us_per_restore_extrapolated": round(wall / len(layers) * case.shape.num_layers * 1e6, 1),
        "checkpoint_write_cpu_s_per_layer": round(write_cpu / len(layers), 3),
        "restore_s_per_layer_in_pool": round(restore_cpu / len(layers), 3),
        "restore_s_one_layer_one_worker": round(one_layer_s, 3),
        "one_worker_GBps": round(per_layer_bytes / one_layer_s / 1e9, 4),
        "cpu_model": _cpu_model(),
    }


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_configs(max_workers: int = 16, sampled_layers: int = 4) -> dict:
    """The oracle timed on every named configuration (``--oracle-configs``),
    one process per (request, layer) job: the one-layer configurations and
    the 32-layer one in full, the 70B-shaped and batched ones on their first
    ``sampled_layers`` layers, extrapolated linearly in layers.  The wall
    estimate assumes the jobs spread evenly over the workers."""
    from paper_2609_26219_amd import workloads as wl

    try:
        n_cpu = len(os.sched_getaffinity(0))
    except AttributeError:
        n_cpu = os.cpu_count() or 1
    workers = max(1, min(max_workers, n_cpu))
    out = {"workers": workers, "cpu_model": _cpu_model()}
    for name in ("tiny", "llama8b_1l", "llama8b_32l", "llama70b", "batched16"):
        case = wl.make_case(name)
        L = case.shape.num_layers
        layers = list(range(L)) if L <= 32 else list(range(sampled_layers))
        if name == "batched16":
            layers = list(range(sampled_layers))
        jobs = [(case, ri, l) for ri in range(len(case.requests)) for l in layers]
        t = time.perf_counter()
        pool = mp.get_context("fork").Pool(min(workers, len(jobs)))  # this mode never touches the GPU
        try:
            times = pool.map(_oracle_layer, jobs)
        finally:
            pool.close()
            pool.join()
        wall_measured = time.perf_counter() - t
        restore_cpu = sum(r for r, _ in times)
        full_cpu = restore_cpu * L / len(layers)
        est_wall = full_cpu / min(workers, len(jobs) * L // len(layers))
        nbytes = case.algorithmic_bytes()["total"]
        out[name] = {
            "requests": len(case.requests),
            "layers_timed": len(layers),
            "layers": L,
            "extrapolated": len(layers) < L,
            "restore_cpu_s_timed": round(restore_cpu, 3),
            "restore_cpu_s_full": round(full_cpu, 3),
            "est_wall_s": round(est_wall, 4),
            "GBps": round(nbytes / est_wall / 1e9, 4),
            "job_mean_s": round(restore_cpu / len(jobs), 4),
            "sample_wall_s_incl_checkpoint_write": round(wall_measured, 2),
        }
        log(f"[bench] oracle {name}: {out[name]['est_wall_s']} s per restore at {workers} workers"
            f"{' (extrapolated)' if len(layers) < L else ''}, {out[name]['GBps']} GB/s")
    return out


def oracle_parity(case, dr, layers) -> dict:
    """Parity of the timed restore with the oracle, on sampled layers of
    request 0 (part of the CPU-baseline leg).  For each sampled layer: the GPU-written
    checkpoint against the quantize oracle's, byte for byte; every restored
    element against the restore oracle's exact value from the oracle's
    checkpoint, in steps of the output format; and, over every layer, each
    element the restore must not write against the cache's pre-fill."""
    import numpy as np

    import oracle
    from oracle import quantize as oq

    s = case.shape
    req = case.requests[0]
    one = dataclasses.replace(req, payload_offset=0, scale_offset=0)
    s1 = dataclasses.replace(s, num_layers=1)
    blocks = oracle.reused_blocks(req)
    layout = oracle.block_layout(req.tags, s.block_tokens, s.num_kv_heads, s.head_dim)
    slots = np.concatenate([oracle.destination_slots(s, req, b) for b in blocks])

    def ordered(bits):
        b = bits.astype(np.int32)
        return np.where(b & 0x8000, -(b & 0x7FFF), b)

    ckpt_bad = n = n_exact = n_near = n_wrong = max_ulp = n_nan = 0
    max_abs_unit = 0.0
    for layer in layers:
        _, kb, vb = case.suffix_bits(0, layer)
        pb, sb = oq.quantize_rows(s, req, kb, vb)
        po, so = case.layer_payload_offset(0, layer), case.layer_scale_offset(0, layer)
        ckpt_bad += int((dr.payload[po:po + pb.size].cpu().numpy() != pb).sum())
        ckpt_bad += int((dr.scales[so:so + sb.size].cpu().numpy().view(np.uint16) != sb.reshape(-1)).sum())
        got = (dr.rows(0, layer, slots), dr.rows(1, layer, slots))
        pos = 0
        for b in blocks:
            _, k, v = oracle.restore_block(pb, sb.reshape(-1), s1, one, 0, b, layout)
            m = k.shape[0]
            for g, exact, slack in ((got[0][pos:pos + m], k, oracle.rotation_slack(k, int(req.delta))),
                                    (got[1][pos:pos + m], v, None)):
                want = oracle.round_to_output(exact, s.out_dtype)
                same, near = oracle.classify_outputs(g, exact, s.out_dtype, slack)
                d = np.abs(ordered(g) - ordered(want))
                n += d.size
                n_exact += int(same.sum())
                n_near += int(near.sum())
                n_wrong += int((~(same | near)).sum())
                max_ulp = max(max_ulp, int(d.max()))
                vals = oracle.output_values(g, s.out_dtype)
                n_nan += int(np.isnan(vals).sum())
                unit = np.abs(exact) < 8.0
                if unit.any():
                    max_abs_unit = max(max_abs_unit, float(np.abs(vals - exact)[unit].max()))
            pos += m
    untouched_bad = dr.untouched_mismatches(oracle.written_slots(s, case.requests))
    return {
        "sample": f"request 0, layers {list(layers)} of {s.num_layers}: {len(blocks)} reused blocks per layer, "
                  f"{n} restored elements; untouched elements checked in all {s.num_layers} layers",
        "checkpoint_byte_mismatches": ckpt_bad,
        "max_ulp": max_ulp,
        "bit_identical_fraction": round(n_exact / max(1, n), 7),
        "near_tie_neighbours": n_near,
        "wrong_elements": n_wrong,
        "rule": "each element is the exactly rounded fp64 oracle value, or the other neighbour of a rounding "
                "midpoint within 2^-23 |x| (+ the rotation slack for keys) of the exact value",
        "max_abs_err_unit_scale": max_abs_unit,
        "nan_outputs": n_nan,
        "untouched_mismatches": int(untouched_bad),
        "pass": bool(ckpt_bad == 0 and n_wrong == 0 and max_ulp <= 1 and n_nan == 0 and untouched_bad == 0),
    }


# ---------------------------------------------------------------------------


# Side measurements first keep the GPU busy this long (untimed, back to
# back).  Measured: after a second or more of idling (drawing inputs on the
# CPU, host-side checks), launches 3-12 of the 8B-shaped checkpoint write run
# 8-22% slower than its steady ~1080 us while the device ramps back up, so a
# fixed count of two warm-up launches left the ramp inside the timed ones.
STEADY_WARM_S = 0.2


def time_launches(torch, launch, n: int, warmup: int, stream, warm_s: float = 0.0):
    """Per-launch durations (ms, sorted) from HIP events on ``stream`` and the
    wall time (s) of the ``n`` timed launches.  ``warmup`` untimed launches
    first, then more until ``warm_s`` seconds have passed (0 for the headline
    step, whose warm-up count the command line fixes)."""
    for i in range(warmup):
        launch(i)
    torch.cuda.synchronize()
    t_warm = time.perf_counter()
    i = warmup
    while time.perf_counter() - t_warm < warm_s:
        for _ in range(8):
            launch(i)
            i += 1
        torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(n):
        ev[i][0].record(stream)
        launch(i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return sorted(a.elapsed_time(b) for a, b in ev), wall


def warm_up(torch, run, min_seconds: float = 0.5, min_calls: int = 2) -> int:
    """Untimed calls for at least ``min_seconds``.  Measured: transfers from a
    newly prepared pinned checkpoint run 20-30% slower for their first ~0.2 s
    (the same calls then settle), so one warm-up call is not enough.  Returns
    the number of calls made."""
    t0 = time.perf_counter()
    n = 0
    while n < min_calls or time.perf_counter() - t0 < min_seconds:
        run()
        torch.cuda.synchronize()
        n += 1
    return n


def host_restore(torch, binding, dr, steps: int, stream):
    """Streamed restore from pinned host memory (pkv_restore_from_host): the
    checkpoint sits in pinned host DRAM; per layer, only reused blocks and the
    layer's scales are copied, overlapped with the previous layer's restore."""
    hp = torch.empty(dr.payload.numel(), dtype=torch.uint8, pin_memory=True)
    hs = torch.empty(dr.scales.numel(), dtype=torch.int16, pin_memory=True)
    hp.copy_(dr.payload)
    hs.copy_(dr.scales)
    torch.cuda.synchronize()
    info = dr.info
    run = lambda: binding.restore_from_host_tensors(dr.plan, hp, hs, dr.payload, dr.scales, dr.k_cache, dr.v_cache,
                                                     stream)
    warm_up(torch, run)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        run()
        b.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)
    avg = sum(ms) / len(ms)
    # zero-copy: the restore kernel reads the pinned checkpoint directly
    zc = lambda: binding.restore_tensors(dr.plan, hp, hs, dr.k_cache, dr.v_cache, stream)
    warm_up(torch, zc)
    zev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in zev:
        a.record(stream)
        zc()
        b.record(stream)
    torch.cuda.synchronize()
    zms = sorted(a.elapsed_time(b) for a, b in zev)
    zavg = sum(zms) / len(zms)
    # practical ceiling: one pinned host -> device copy of the same byte count
    n = int(info["host_copy_bytes"])
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    src = hp[:n] if hp.numel() >= n else torch.empty(n, dtype=torch.uint8, pin_memory=True)
    warm_up(torch, lambda: dst.copy_(src, non_blocking=True))
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(3):
        dst.copy_(src, non_blocking=True)
    b.record(stream)
    torch.cuda.synchronize()
    copy_gbps = n / (a.elapsed_time(b) / 3 * 1e-3) / 1e9
    del dst
    need = int(info["bytes_read"])  # reused blocks' payload and scales: what must cross the link
    achieved = need / (avg * 1e-3) / 1e9
    full = dr.payload.numel() + 2 * dr.scales.numel()
    zachieved = need / (zavg * 1e-3) / 1e9
    log(f"[bench] streamed restore from host: {avg:.2f} ms, {n / (avg * 1e-3) / 1e9:.1f} GB/s copied over the host "
        f"link, {achieved:.1f} GB/s of reused-block bytes (one plain pinned copy of the same bytes: {copy_gbps:.1f} GB/s); "
        f"zero-copy restore {zavg:.2f} ms, {zachieved:.1f} GB/s")
    return {
        "what": "pkv_restore_from_host: per layer, reused blocks' payload ranges and the layer's scales copied "
                "from pinned host memory on a copy stream, each layer's restore enqueued behind its copies",
        "fetch_and_dequant_ms": round(avg, 3),
        "ms_p10_p50_p90": [round(ms[int(q * (len(ms) - 1))], 3) for q in (0.1, 0.5, 0.9)],
        "steps": len(ms),
        "algorithmic_bytes": need,
        "bytes_copied": n,
        "checkpoint_bytes": full,
        "copies": int(info["host_copies"]),
        "copied_GBps": round(n / (avg * 1e-3) / 1e9, 2),
        "roofline": {
            "bound": "pcie",
            "achieved": round(achieved, 2),
            "peak": PCIE_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / PCIE_PEAK_GBPS, 4),
            "traffic": None,
        },
        "plain_pinned_copy_GBps": round(copy_gbps, 2),
        "zero_copy": {
            "what": "pkv_restore with the checkpoint in pinned host memory: the kernel reads only the reused "
                    "blocks over the host link, one launch",
            "ms": round(zavg, 3),
            "ms_p10_p50_p90": [round(zms[int(q * (len(zms) - 1))], 3) for q in (0.1, 0.5, 0.9)],
            "GBps": round(zachieved, 2),
            "frac_of_pcie_peak": round(zachieved / PCIE_PEAK_GBPS, 4),
        },
        "copied_frac_of_plain_copy": round(n / (avg * 1e-3) / 1e9 / copy_gbps, 4),
    }


def checkpoint_to_host(torch, binding, ck, old, stream, steps: int):
    """The checkpoint write straight into pinned host memory (where the paper
    keeps checkpoints): the kernel stores the checkpoint over the host link,
    no staging copy.  Its output is checked against the device-written one."""
    hp = torch.empty(ck.payload.numel(), dtype=torch.uint8, pin_memory=True)
    hs = torch.empty(ck.scales.numel(), dtype=torch.int16, pin_memory=True)
    run = lambda i: binding.quantize_gather_tensors(ck.plan, old.k, old.v, hp, hs, stream)
    ms, _ = time_launches(torch, run, steps, 2, stream, STEADY_WARM_S)
    avg = sum(ms) / len(ms)
    same = bool(torch.equal(hp.to(ck.payload.device), ck.payload) and torch.equal(hs.to(ck.scales.device), ck.scales))
    written = int(ck.info["bytes_written"])
    log(f"[bench] checkpoint write into pinned host memory: {avg:.2f} ms, {written / (avg * 1e-3) / 1e9:.1f} GB/s "
        f"over the host link, identical to the device-written checkpoint: {same}")
    return {
        "what": "the same pkv_quantize_gather launch with payload and scales in pinned host memory: the kernel "
                "writes the checkpoint over the host link",
        "ms": round(avg, 3),
        "ms_p10_p50_p90": [round(ms[int(q * (len(ms) - 1))], 3) for q in (0.1, 0.5, 0.9)],
        "launches": len(ms),
        "bytes_written_over_link": written,
        "GBps": round(written / (avg * 1e-3) / 1e9, 2),
        "frac_of_pcie_peak": round(written / (avg * 1e-3) / 1e9 / PCIE_PEAK_GBPS, 4),
        "identical_to_device_write": same,
    }


def planner_timing(binding, case, reps: int = 20):
    """Resume planner (pkv_plan_repair, host C++) on each request of the
    workload: dirty window d_hat = 12% of the suffix, kappa = 1.5%, stored
    importance drawn log-normal and correlated within 32-token spans (a
    span-level factor of sigma 2 times a token-level one of sigma 0.5:
    attention mass concentrates on spans), seeded; only its ranking matters."""
    import numpy as np

    from oracle import planner as op

    rng = np.random.default_rng(case.seed + 9)
    rows = []
    t_lib = t_orc = 0.0
    for r in case.requests:
        N, B = int(r.suffix_tokens), int(case.shape.block_tokens)
        span = rng.normal(0.0, 2.0, size=-(-N // 32)).repeat(32)[:N]
        imp = np.exp(span + rng.normal(0.0, 0.5, size=N)).astype(np.float32)
        imp /= imp.sum()
        d_hat = int(0.12 * N)
        t = time.perf_counter()
        for _ in range(reps):
            mask, h = binding.pkv_plan_repair(N, B, d_hat, imp, 0.015)
        t_lib += (time.perf_counter() - t) / reps
        t = time.perf_counter()
        want, _ = op.repair_mask(N, B, d_hat, imp, 0.015)
        t_orc += time.perf_counter() - t
        assert mask.tolist() == want
        rows.append((N, int(mask.sum()), len(mask), h))
    n_blocks = sum(x[2] for x in rows)
    return {
        "what": "pkv_plan_repair on the host: D = first 12% of the suffix (Eq. 9), H = top 1.5% of the rest by "
                "stored importance (Eq. 11), R = BlockRound(D u H) (Eq. 12)",
        "requests": len(rows),
        "us_per_request": round(t_lib / len(rows) * 1e6, 1),
        "oracle_us_per_request": round(t_orc / len(rows) * 1e6, 1),
        "repair_blocks_fraction": round(sum(x[1] for x in rows) / max(1, n_blocks), 4),
        "nonlocal_tokens": sum(x[3] for x in rows),
    }


REPRESENTATIONS = (("FP16", 0), ("INT8 (K8V8)", 1), ("K8V4", 2), ("INT4 (K4V4)", 3), ("mixed (workload tags)", None))


def representations(torch, binding, wl, case, old, steps: int, host_steps: int, stream):
    """The representation axis of the transport ablation: the same suffix,
    repair set and old caches, checkpointed uniformly in one representation
    (or with the workload's per-block tags), then restored from HBM and
    streamed from pinned host memory."""
    import dataclasses

    import numpy as np

    from paper_2609_26219_amd.device import DeviceCheckpoint, DeviceRestore

    rows = []
    for label, tag in REPRESENTATIONS:
        reqs = [dataclasses.replace(r, tags=np.full_like(r.tags, tag)) if tag is not None else r
                for r in case.requests]
        c = wl.Case(case.name, case.shape, [dataclasses.replace(r) for r in reqs], case.seed, case.distinct_layers,
                    case.outlier_pairs)
        ck = DeviceCheckpoint(c, old)
        ck.write(stream)
        torch.cuda.synchronize()
        dr = DeviceRestore(c, checkpoint=(ck.payload, ck.scales))
        del ck
        info = dr.info
        nbytes = info["bytes_read"] + info["bytes_written"]
        ms, _ = time_launches(torch, lambda i: dr.run(stream), steps, 2, stream, STEADY_WARM_S)
        avg = sum(ms) / len(ms)
        host = host_restore(torch, binding, dr, host_steps, stream)
        rows.append({
            "representation": label,
            "checkpoint_bytes": int(c.payload_nbytes + 2 * c.scale_elems),
            "restore_bytes_read": int(info["bytes_read"]),
            "restore_us": round(avg * 1e3, 1),
            "restore_GBps": round(nbytes / (avg * 1e-3) / 1e9, 1),
            "pct_hbm_peak": round(100 * nbytes / (avg * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
            "from_host_ms": host["fetch_and_dequant_ms"],
            "from_host_GBps": host["roofline"]["achieved"],
            "zero_copy_ms": host["zero_copy"]["ms"],
            "zero_copy_GBps": host["zero_copy"]["GBps"],
        })
        log(f"[bench] {label}: checkpoint {rows[-1]['checkpoint_bytes'] / 2**20:.1f} MiB, restore "
            f"{rows[-1]['restore_us']} us ({rows[-1]['pct_hbm_peak']}% HBM), from host {rows[-1]['from_host_ms']} ms "
            f"(DMA), {rows[-1]['zero_copy_ms']} ms (zero-copy)")
        del dr
        torch.cuda.empty_cache()
    return rows


def other_layout(torch, wl, case, dr, stream, steps: int = 20):
    """The same restore (same checkpoint, plan inputs and page tables) into
    caches of the other layout, for comparison."""
    from paper_2609_26219_amd.device import DeviceRestore

    other = wl.KV_SEPARATE if case.shape.kv_layout == wl.KV_PAIRED else wl.KV_PAIRED
    c = wl.Case(case.name, dataclasses.replace(case.shape, kv_layout=other), case.requests, case.seed,
                case.distinct_layers, case.outlier_pairs)
    d2 = DeviceRestore(c, checkpoint=(dr.payload, dr.scales))
    info = d2.info
    nbytes = info["bytes_read"] + info["bytes_written"]
    ms, _ = time_launches(torch, lambda i: d2.run(stream), steps, 3, stream, STEADY_WARM_S)
    avg = sum(ms) / len(ms)
    del d2
    torch.cuda.empty_cache()
    name = "paired" if other == wl.KV_PAIRED else "separate"
    log(f"[bench] {name} caches: {avg * 1e3:.1f} us ({100 * nbytes / (avg * 1e-3) / 1e9 / HBM_PEAK_GBPS:.2f}% HBM)")
    return {
        "kv_layout": KV_LAYOUT_TEXT[name],
        "us_per_restore": round(avg * 1e3, 1),
        "us_p10_p50_p90": [round(ms[int(q * (len(ms) - 1))] * 1e3, 1) for q in (0.1, 0.5, 0.9)],
        "GBps": round(nbytes / (avg * 1e-3) / 1e9, 1),
        "pct_hbm_peak": round(100 * nbytes / (avg * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
    }


def small_restores(torch, wl, layout: int, stream, n: int = 50):
    """The configurations whose working set fits the 256 MB MALL (Tiny, one
    8B-shaped layer): per-launch time warm (back to back) and cold (a 1 GiB
    scratch write before each launch, outside its events, so no byte of the
    restore's inputs or outputs is left in the MALL)."""
    from paper_2609_26219_amd.device import DeviceRestore

    scratch = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    out = {}
    for name in ("tiny", "llama8b_1l"):
        case = wl.make_case(name)
        case.shape = dataclasses.replace(case.shape, kv_layout=layout)
        dr = DeviceRestore(case)
        info = dr.info
        nbytes = info["bytes_read"] + info["bytes_written"]
        warm, _ = time_launches(torch, lambda i: dr.run(stream), n, 5, stream, STEADY_WARM_S)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for i in range(n):
            scratch.fill_(i & 0xFF)
            ev[i][0].record(stream)
            dr.run(stream)
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        cold = sorted(a.elapsed_time(b) for a, b in ev)
        row = {"algorithmic_bytes": nbytes, "launches": n}
        for label, ms in (("warm", warm), ("cold", cold)):
            avg = sum(ms) / len(ms)
            row[f"us_{label}"] = round(avg * 1e3, 2)
            row[f"us_{label}_p50"] = round(ms[len(ms) // 2] * 1e3, 2)
            row[f"GBps_{label}"] = round(nbytes / (avg * 1e-3) / 1e9, 1)
        log(f"[bench] {name}: {row['us_warm']} us warm, {row['us_cold']} us cold")
        out[name] = row
        del dr
    del scratch
    torch.cuda.empty_cache()
    return out


def copy_reference(torch, nbytes: int = 4 << 30, reps: int = 10):
    """Plain device-to-device copy (read + write bytes / time): the practical ceiling."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    torch.cuda.empty_cache()
    return round(2 * nbytes / (ms * 1e-3) / 1e9, 1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama8b_32l", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--int4", default="K8V4", choices=["K8V4", "K4V4"],
                    help="representation of the int4 tag: K8V4 (the paper's tier) or uniform K4V4")
    ap.add_argument("--kv-layout", default="paired", choices=["paired", "separate"],
                    help="paged cache layout: one [L][pool_pages][2][P][H][D] cache (paired) or two caches")
    ap.add_argument("--sets", type=int, default=2, help="buffer sets cycled between steps")
    ap.add_argument("--write-steps", type=int, default=10, help="timed checkpoint-write launches")
    ap.add_argument("--host-steps", type=int, default=10, help="timed streamed restores from pinned host memory")
    ap.add_argument("--no-representations", action="store_true",
                    help="skip the uniform-representation comparison (FP16 / K8V8 / K8V4 / K4V4 / mixed)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ref", action="store_true")
    ap.add_argument("--no-other-layout", action="store_true", help="skip timing the restore on the other cache layout")
    ap.add_argument("--no-small", action="store_true", help="skip the warm/cold Tiny and one-layer restores")
    ap.add_argument("--oracle-configs", action="store_true",
                    help="only time the CPU oracle on every named configuration and print that as JSON")
    args = ap.parse_args()

    if args.oracle_configs:
        print(json.dumps({"cpu_oracle_configs": oracle_configs()}), flush=True)
        return

    if args.gpus != 1:
        print(f"bench.py: the restore is measured on one GPU; --gpus {args.gpus} is not supported "
              f"(the restore shards by request, layer or KV head with no exchange step).", file=sys.stderr)
        sys.exit(2)

    # Worker processes (row draws, the CPU oracle) are forked now, before
    # anything touches the GPU, and joined at the end.
    from paper_2609_26219_amd import device
    from paper_2609_26219_amd import workloads as wl

    n_workers = wl.default_workers()
    pool = device.start_workers(n_workers)
    try:
        run(args, pool, n_workers)
    finally:
        device.stop_workers()


def run(args, pool, n_workers):
    import torch

    from paper_2609_26219_amd import binding
    from paper_2609_26219_amd import workloads as wl
    from paper_2609_26219_amd.device import DeviceCheckpoint, DeviceRestore, OldCaches

    binding.load()
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    int4_tag = wl.TAG_K8V4 if args.int4 == "K8V4" else wl.TAG_K4V4
    t = time.perf_counter()
    case = wl.make_case(args.workload, int4_tag=int4_tag)
    layout = wl.KV_PAIRED if args.kv_layout == "paired" else wl.KV_SEPARATE
    case.shape = dataclasses.replace(case.shape, kv_layout=layout)
    stream = torch.cuda.current_stream()
    layerwise = args.workload in LAYERWISE
    if layerwise:
        args.sets, args.host_steps = 1, 0
        args.no_representations = args.no_other_layout = True
        old = None
        sets = [DeviceRestore(case)]
        log(f"[bench] wrote the {args.workload} checkpoint layer by layer in {time.perf_counter() - t:.1f} s")
        checkpoint_write = None
    else:
        old = OldCaches(case)
        log(f"[bench] drew {args.workload} old caches in {time.perf_counter() - t:.1f} s")
        # Checkpoint write (offload side): every layer, every block, one launch.
        ck = DeviceCheckpoint(case, old)
        w_info = ck.info
        w_bytes = w_info["bytes_read"] + w_info["bytes_written"]
        w_ms, _ = time_launches(torch, lambda i: ck.write(stream), args.write_steps, 2, stream, STEADY_WARM_S)
        w_avg = sum(w_ms) / len(w_ms)
        w_achieved = w_bytes / (w_avg * 1e-3) / 1e9
        log(f"[bench] checkpoint write avg {w_avg * 1e3:.1f} us, {w_achieved:.0f} GB/s")
        checkpoint_write = {
            "what": "pkv_quantize_gather of every block of every layer from the old paged caches "
                    "(the offload side that produces the restored checkpoint), one launch",
            "us": round(w_avg * 1e3, 1),
            "us_p10_p50_p90": [round(w_ms[int(q * (len(w_ms) - 1))] * 1e3, 1) for q in (0.1, 0.5, 0.9)],
            "launches": len(w_ms),
            "algorithmic_bytes": w_bytes,
            "bytes_read": w_info["bytes_read"],
            "bytes_written": w_info["bytes_written"],
            "roofline": {
                "bound": "hbm",
                "achieved": round(w_achieved, 1),
                "peak": HBM_PEAK_GBPS,
                "unit": "GB/s",
                "frac": round(w_achieved / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(args.workload, args.int4, args.kv_layout, "gather_tile_kernel",
                                            GATHER_SRC),
            },
        }
        if args.host_steps > 0:
            checkpoint_write["to_pinned_host"] = checkpoint_to_host(torch, binding, ck, old, stream, args.host_steps)
        ck.old = None
        sets = [DeviceRestore(case, checkpoint=(ck.payload, ck.scales)) for _ in range(max(1, args.sets))]
        del ck
    torch.cuda.empty_cache()
    info = sets[0].info
    nbytes = info["bytes_read"] + info["bytes_written"]
    alg = case.algorithmic_bytes()
    assert nbytes == alg["total"], (nbytes, alg)
    log(f"[bench] {len(sets)} buffer set(s) ready; {info['num_units']} workgroups, {nbytes / 1e9:.3f} GB per step")

    kern_ms, wall = time_launches(torch, lambda i: sets[i % len(sets)].run(stream), args.steps, args.warmup, stream)
    kern_avg_ms = sum(kern_ms) / len(kern_ms)
    ms_per_step = wall * 1e3 / args.steps
    log(f"[bench] kernel avg {kern_avg_ms * 1e3:.1f} us (median {kern_ms[len(kern_ms) // 2] * 1e3:.1f}), "
        f"wall {ms_per_step * 1e3:.1f} us/step")

    achieved = nbytes / (kern_avg_ms * 1e-3) / 1e9
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f64",
        "data": "synthetic",
        "config": {
            "workload": WORKLOAD_TEXT[args.workload],
            "name": args.workload,
            "int4_tag": args.int4,
            "requests": len(case.requests),
            "restored_tokens": case.restored_tokens(),
            "algorithmic_bytes": nbytes,
            "bytes_read": info["bytes_read"],
            "bytes_written": info["bytes_written"],
            "buffer_sets": len(sets),
            "kv_layout": KV_LAYOUT_TEXT[args.kv_layout],
        },
        "us_per_restore": round(kern_avg_ms * 1e3, 1),
        "us_per_restore_p10_p50_p90": [round(kern_ms[int(q * (len(kern_ms) - 1))] * 1e3, 1) for q in (0.1, 0.5, 0.9)],
        "pct_hbm_peak": round(100 * achieved / HBM_PEAK_GBPS, 2),
        "restored_tokens_per_s": round(case.restored_tokens() / (kern_avg_ms * 1e-3), 1),
        "output_GBps": round(info["bytes_written"] / (kern_avg_ms * 1e-3) / 1e9, 1),
        "roofline": {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": measured_traffic(args.workload, args.int4, args.kv_layout),
        },
        "checkpoint_write": checkpoint_write if checkpoint_write is not None else
        "not timed: this workload's old caches of all layers do not fit beside its pool, so its checkpoint is "
        "written layer by layer",
    }
    parity = None
    if not args.no_cpu_baseline:
        parity = oracle_parity(case, sets[0], (0, case.shape.num_layers - 1))
        log(f"[bench] oracle parity: max ulp {parity['max_ulp']}, bit-identical {parity['bit_identical_fraction']}, "
            f"near-tie neighbours {parity['near_tie_neighbours']}, wrong {parity['wrong_elements']}, "
            f"checkpoint mismatches {parity['checkpoint_byte_mismatches']}, untouched mismatches "
            f"{parity['untouched_mismatches']}")
    if not args.no_other_layout:
        out["other_kv_layout"] = other_layout(torch, wl, case, sets[0], stream)
    if args.host_steps > 0:
        out["host_restore"] = host_restore(torch, binding, sets[0], args.host_steps, stream)
    if not args.no_small:
        out["small_restores"] = small_restores(torch, wl, layout, stream)
    if not args.no_representations:
        del sets[1:]
        torch.cuda.empty_cache()
        out["representations"] = representations(torch, binding, wl, case, old, 10, max(1, min(args.host_steps, 3)),
                                                  stream)
    del old
    torch.cuda.empty_cache()
    out["planner"] = planner_timing(binding, case)
    log(f"[bench] planner: {out['planner']['us_per_request']} us per request "
        f"(oracle {out['planner']['oracle_us_per_request']} us), repair fraction {out['planner']['repair_blocks_fraction']}")
    if not args.no_copy_ref:
        del sets
        torch.cuda.empty_cache()
        out["copy_ref_GBps"] = copy_reference(torch)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(case, pool, n_workers)
        out["cpu_baseline"]["oracle_parity"] = parity
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
