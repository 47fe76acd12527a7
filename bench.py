#!/usr/bin/env python3
"""Fork-decode attention + prefix KV import on one MI355X.

One step = restore a trace's prefix KV blocks from a contiguous staging copy
into the paged pool (specgen_kv_import), then one decode step of fork-decode
attention for all forks (specgen_fork_decode_attn: split partial kernel, then
the log-sum-exp merge).  Inputs are seeded synthetic tensors already resident
in HBM.  R replicas of the pool/q rotate so that every step reads data no
cache level still holds (a replica is far larger than the 256 MB MALL): step k
imports into replica k % R and attends over replica (k+1) % R, whose prefix
was restored R-1 steps earlier.

Prints one JSON line.  `value` is the attention call's achieved HBM rate in
GB/s: algorithmic bytes (each valid prefix token's K/V once per kv head, each
suffix token's K/V once, q in, out/lse out, index arrays) over the median
attention time measured with HIP events on the launch stream, cold (the
replica it reads was last touched three steps earlier).  Beside it: the same
call warm (one replica, repeated), and replayed from HIP graphs (one captured
call per replica, replayed in rotation, so still cold); the partial kernel's
own time (the roofline figure); the streaming read and copy rates a plain
kernel reaches on this GPU (the practical ceilings); the export of the same
prefix blocks (specgen_kv_export) and the per-step append of every fork's next
token (specgen_kv_append), timed on their own; and the oracle on the host's
cores (all of them, and one).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "fork-decode attention achieved HBM GB/s (% of peak) + fork-tokens/s at P=32k,F=16"
HBM_PEAK_GBPS = 8000.0
SPIN_CYCLES = 40_000_000   # GPU clock cycles of the spin that runs ahead of the timed steps


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix peak of the MI355X


# the partial kernel of the MFMA path (bf16 or E4M3 KV), and the sources it includes
def partial_kernel(D: int, fp8: bool, qk8: bool = False) -> str:
    return f"attn_bf16_kernel<{D}, {'true' if fp8 else 'false'}, {'true' if qk8 else 'false'}>"


PARTIAL_SOURCES = ("attn_bf16.hip", "worker.h", "common.h", "plan.h", "lds_layout.h")


def source_hash() -> str:
    h = hashlib.sha256()
    for f in PARTIAL_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_17518_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload: str):
    """HBM traffic of the partial kernel from committed rocprofv3 counter runs,
    only if they were taken on the current kernel source."""
    p = os.path.join(ROOT, "profiles", f"traffic_partials_{workload}.json")
    if not os.path.exists(p):
        return None
    with open(p) as fh:
        d = json.load(fh)
    if d.get("source_hash") != source_hash():
        return None
    return d.get("traffic_bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(batch, target_s: float, q_len=None, step_bytes=None):
    """The fp64 oracle on the same workload on this host's cores: whole decode
    steps (every fork and q head; every query with q_len) repeated until about
    target_s of CPU work on all threads; then one thread on a sample of rows
    (about target_s / 3), scaled to a whole step by the fraction of rows."""
    import oracle
    run = (lambda: oracle.fork_decode_attn(batch)) if q_len is None else (lambda: oracle.fork_prefill_attn(batch, q_len))
    t0 = time.perf_counter()
    run()
    reps = 1
    while time.perf_counter() - t0 < target_s and reps < 64:
        run()
        reps += 1
    dt = time.perf_counter() - t0
    step_s = dt / reps
    step_bytes = batch.algorithmic_bytes() if step_bytes is None else step_bytes
    # one thread, on the first rows of the step (rows cost alike: every row
    # of a fork reads the same keys)
    cores = oracle.max_threads()
    nq = batch.num_forks if q_len is None else int(np.sum(q_len))
    total_rows = nq * batch.num_q_heads
    n1 = max(1, min(total_rows, int(total_rows * (target_s / 3) / (step_s * cores))))
    rows = np.stack(np.divmod(np.arange(n1), batch.num_q_heads), axis=1).astype(np.int32)
    t1 = time.perf_counter()
    if q_len is None:
        oracle.fork_decode_attn(batch, rows=rows, nthreads=1)
    else:
        oracle.fork_prefill_attn(batch, q_len, rows=rows, nthreads=1)
    dt1 = time.perf_counter() - t1
    step1_s = dt1 * total_rows / n1
    oracle.fork_decode_attn(batch, rows=rows[:1], nthreads=cores)   # back to every thread
    return {"value": round(step_bytes / step_s / 1e9, 4), "unit": "GB/s",
            "fork_tokens_per_s": round(batch.num_forks / step_s, 3), "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(),
            "one_thread": {"value": round(step_bytes / step1_s / 1e9, 5), "unit": "GB/s",
                           "sample": f"{n1} of {total_rows} rows on 1 thread in {dt1:.1f} s, scaled to the step"},
            "sample": f"{reps} whole decode steps ({batch.num_forks} forks x {batch.num_q_heads} q heads) of the same "
                      f"workload, fp64 C oracle, {dt:.1f} s; GB/s = step algorithmic bytes / mean step time"}


def stream_ceilings(dev, stream, reps: int = 10, batch=None, fb=None):
    """Streaming read (1 GiB) and copy (512 MiB -> 512 MiB) rates of the plain
    probe kernels (libspecgen_probe.so), and the rate of the bf16 partial
    kernel's own access pattern with no arithmetic (the slice-ring probe: 4 KiB
    kv-head slices of random pool blocks through the same eight-wave LDS-DMA
    ring, 1 GiB; and, for a bf16 head_dim-128 workload, the workload's own
    first prefix on 256 workgroups as the partial kernel launches them):
    medians over `reps` launches, each timed with HIP events on the launch
    stream."""
    import ctypes as C
    import torch
    from paper_2606_17518_amd.build import PROBE_LIB_PATH
    lib = C.CDLL(PROBE_LIB_PATH)
    lib.specgen_probe_stream_read.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
    lib.specgen_probe_stream_copy.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]
    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.int32, device=dev).random_(0, 1 << 30)
    half = torch.empty(nbytes // 8, dtype=torch.int32, device=dev)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    sp = C.c_void_p(stream.cuda_stream)

    def timed(fn):
        ms = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            assert fn() == 0
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return float(np.median(ms))
    read_ms = timed(lambda: lib.specgen_probe_stream_read(src.data_ptr(), nbytes, sink.data_ptr(), sp))
    copy_ms = timed(lambda: lib.specgen_probe_stream_copy(half.data_ptr(), src.data_ptr(), nbytes // 2, sp))
    out = {"read_gbps": round(nbytes / (read_ms / 1e3) / 1e9, 1),
           "copy_gbps": round(nbytes / (copy_ms / 1e3) / 1e9, 1)}
    # slice ring over the 1 GiB buffer as two 512 MiB pools of 16384 blocks x 8 kv heads
    ring = lib.specgen_probe_slice_ring
    ring.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int, C.c_void_p, C.c_int, C.c_int, C.c_void_p,
                     C.c_void_p]
    hkv, nblk = 8, (nbytes // 2) // (8 * 4096)
    tph = nblk // 4
    perm = torch.from_numpy(np.random.default_rng(7).permutation(nblk).astype(np.int32)).to(dev)
    kp, vp = src.data_ptr(), src.data_ptr() + nbytes // 2
    ring_ms = timed(lambda: ring(kp, vp, nblk, hkv, perm.data_ptr(), tph, 256, sink.data_ptr(), sp))
    out["slice_ring_gbps"] = round(hkv * tph * 32768 / (ring_ms / 1e3) / 1e9, 1)
    note = ("plain nontemporal 16-byte streams over every CU: 1 GiB read; 512 MiB copied (1 GiB of traffic); "
            "slice ring: the bf16 partial kernel's tiles (4 KiB K and V slices of one kv head from each of four "
            "random 16-token blocks per 32 KiB tile, eight waves, four LDS stages, LDS-DMA) with no arithmetic, "
            "8 kv heads x 4096 tiles = 1 GiB on 256 workgroups")
    if batch is not None and fb and batch.kv_dtype == "bf16" and batch.head_dim == 128:
        P0 = int(batch.prefix_len[0])
        tiles = -(-P0 // 64)
        o = int(batch.prefix_table_off[0])
        ids = np.asarray(batch.prefix_table[o:o + -(-P0 // 16)], np.int32)
        tab = np.concatenate([ids, np.full(4 * tiles - ids.size, ids[-1], np.int32)])
        tab_d = torch.from_numpy(tab).to(dev)
        turn = [0]

        def prefix_ring():   # the replicas in rotation, as the timed steps read them
            r = fb[turn[0] % len(fb)]
            turn[0] += 1
            return ring(r.k_pool.data_ptr(), r.v_pool.data_ptr(), batch.num_blocks, batch.num_kv_heads,
                        tab_d.data_ptr(), tiles, 256, sink.data_ptr(), sp)
        pms = timed(prefix_ring)
        out["slice_ring_prefix_gbps"] = round(batch.num_kv_heads * tiles * 32768 / (pms / 1e3) / 1e9, 1)
        out["slice_ring_prefix_us"] = round(pms * 1e3, 2)
        note += (f"; slice_ring_prefix: the same ring over trace 0's {P0}-token prefix in this workload's pools "
                 f"({batch.num_kv_heads} kv heads x {tiles} tiles; the replicas in rotation), launch and ramp "
                 f"included")
    out["note"] = note + "; median of 10 launches between HIP events"
    del src, half
    return out


def timeline_report(args, b, step, q_len):
    """Per-workgroup timeline of the partial kernel (libspecgen_timeline.so):
    `warmup` steps, then `steps` steps each read back on its own (stamps
    cleared before it; the attention call queued behind the step's import as
    in the timed run).  Prints medians over the steps of per-step percentiles
    over the workgroups, in microseconds from the first workgroup's start."""
    import ctypes as C
    import torch
    from paper_2606_17518_amd import binding
    T = binding.timeline_lib()
    W, S = C.c_int(0), C.c_int(0)
    assert T.specgen_timeline_shape(C.byref(W), C.byref(S)) == 0
    W, S = W.value, S.value
    stamps = np.zeros((W, S), np.uint64)
    kinds = np.zeros((W, S), np.int32)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for k in range(args.warmup):
        step(k, evs, q_len is None)
    torch.cuda.synchronize()
    rows = []
    for k in range(args.steps):
        assert T.specgen_timeline_clear() == 0
        step(args.warmup + k, evs, q_len is None)
        torch.cuda.synchronize()
        assert T.specgen_timeline_read(stamps.ctypes.data, kinds.ctypes.data) == 0
        live = np.nonzero(stamps[:, 0])[0]
        if live.size == 0:
            print("no workgroup of the MFMA partial kernel ran (the dot path is not stamped)")
            return
        st = stamps[live].astype(np.int64)
        kd = kinds[live]
        t0 = st[:, 0].min()
        us = lambda col: (st[:, col] - t0) * 0.01   # 100 MHz clock
        end = us(S - 1)
        nslot = kd[:, S - 1]
        inter = {-1: [], 0: [], 1: []}
        last = []
        nq = np.zeros(len(live), np.int32)     # q slots: items (or 128-row halves) the worker starts
        nsuf = np.zeros(len(live), np.int32)   # suffix tiles
        for i in range(len(live)):
            n = min(int(nslot[i]), S - 5)
            ts = (st[i, 4:4 + n] - t0) * 0.01
            for s in range(1, n):
                inter[int(kd[i, 4 + s - 1])].append(ts[s] - ts[s - 1])
            if 0 < nslot[i] <= S - 5:   # the whole range was stamped
                last.append(end[i] - ts[n - 1])
            nq[i] = int(np.sum(kd[i, 4:4 + n] == -1))
            nsuf[i] = int(np.sum(kd[i, 4:4 + n] == 1))
        xcd = [float(np.median(end[live % 8 == x])) if np.any(live % 8 == x) else float("nan") for x in range(8)]
        by_q = {q: float(np.median(end[nq == q])) if np.any(nq == q) else float("nan") for q in (1, 2, 3)}
        rows.append({
            "workers": len(live), "start_max": us(0).max(), "plan_p50": np.median(us(1)),
            "walk_p50": np.median(us(2)), "walk_max": us(2).max(),
            "first_slots_issued_p50": np.median(us(3)[nslot > 0]) if np.any(nslot > 0) else float("nan"),
            "slot0_p50": np.median(us(4)), "slot0_max": us(4).max(),
            "end_min": end.min(), "end_p50": np.median(end), "end_max": end.max(),
            "slots_p50": np.median(nslot), "slots_max": nslot.max(),
            "q_slot_interval_p50": np.median(inter[-1]) if inter[-1] else float("nan"),
            "prefix_tile_interval_p50": np.median(inter[0]) if inter[0] else float("nan"),
            "prefix_tile_interval_p90": np.percentile(inter[0], 90) if inter[0] else float("nan"),
            "suffix_tile_interval_p50": np.median(inter[1]) if inter[1] else float("nan"),
            "last_slot_to_end_p50": np.median(last) if last else float("nan"),
            **{f"end_p50_xcd{x}": xcd[x] for x in range(8)},
            **{f"end_p50_workers_with_{q}_q_slots": by_q[q] for q in (1, 2, 3)},
            "end_p50_workers_with_suffix_tiles": float(np.median(end[nsuf > 0])) if np.any(nsuf > 0) else float("nan"),
            "end_p50_workers_without": float(np.median(end[nsuf == 0])) if np.any(nsuf == 0) else float("nan"),
        })
    print(f"timeline of the partial kernel, {args.workload}: medians over {args.steps} steps of per-step figures "
          f"(us from the first workgroup's start; stamps of thread 0 of each workgroup)")
    for key in rows[0]:
        v = float(np.nanmedian([r[key] for r in rows])) if any(np.isfinite(r[key]) for r in rows) else float("nan")
        print(f"  {key:36s} {v:9.2f}")


def pct(a, q):
    return round(float(np.percentile(a, q)) * 1e3, 2)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="trace_p32k_f16")
    ap.add_argument("--replicas", type=int, default=4)
    ap.add_argument("--path", default="auto", choices=["auto", "mfma", "dot"])
    ap.add_argument("--fp8-scores", action="store_true",
                    help="E4M3 KV: scores on the fp8 matrix cores (SPECGEN_FLAG_FP8_SCORES)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--timeline", action="store_true",
                    help="instead of the JSON line: run the steps on libspecgen_timeline.so and print the partial "
                         "kernel's per-workgroup timeline (medians over --steps steps)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the fork-decode path here has no multi-GPU part "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_17518_amd as sg
    import synth
    if args.timeline:   # every library call of the run goes to the stamping build
        from paper_2606_17518_amd import binding
        binding._lib = binding.timeline_lib()

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    spec = synth.WORKLOADS[args.workload]
    log(f"generating {args.workload}")
    b = synth.workload(args.workload)
    prefill_q = spec.get("prefill_q")
    q_len = None
    if prefill_q:   # multi-token prefill: every fork's last prefill_q suffix tokens are queries
        q_len = np.full(b.num_forks, prefill_q, np.int32)
        b = synth.with_prefill_queries(b, q_len, seed=1)
    do_import = spec.get("import_prefix", False)
    R = max(2, args.replicas)
    log(f"uploading {R} replicas")
    reps = []
    for r in range(R):
        fb = sg.ForkBatchTensors.from_numpy(b, dev, args.path,
                                            flags=sg.SPECGEN_FLAG_FP8_SCORES if args.fp8_scores else 0)
        if r > 0:   # index arrays are shared; only q and the pools are replicated
            for name in ("fork_off", "prefix_len", "prefix_table_off", "prefix_table", "suffix_len",
                         "suffix_table_off", "suffix_table"):
                setattr(fb, name, getattr(reps[0], name))
        reps.append(fb)
    N, Hq, D = b.num_forks, b.num_q_heads, b.head_dim
    Q = N if q_len is None else int(q_len.sum())   # query rows per head
    out = torch.empty((Q, Hq, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((Q, Hq), dtype=torch.float32, device=dev)
    ws = sg.alloc_workspace(reps[0]) if q_len is None else sg.alloc_prefill_workspace(reps[0], q_len)
    stream = torch.cuda.current_stream()

    imp = None
    if do_import:
        ks, vs, ids, kss, vss = synth.prefix_import_from_batch(b, 0)
        bb = b.block_bytes()
        ids_d = torch.from_numpy(ids).to(dev)
        imp = []
        for fb in reps:
            tensors = [(fb.k_pool, torch.from_numpy(ks.reshape(-1).view(np.uint8)).to(dev), bb),
                       (fb.v_pool, torch.from_numpy(vs.reshape(-1).view(np.uint8)).to(dev), bb)]
            if kss is not None:
                tensors += [(fb.k_scale, torch.from_numpy(kss).to(dev), 4), (fb.v_scale, torch.from_numpy(vss).to(dev), 4)]
            imp.append(tensors)
            # poison the destination blocks, restore them, and check the restore once
            fb.k_pool.view(b.num_blocks, -1)[ids_d.long()] = -1
            fb.v_pool.view(b.num_blocks, -1)[ids_d.long()] = -1
            sg.specgen_kv_import(tensors, ids_d, b.num_blocks)
        torch.cuda.synchronize()
        ref_k = torch.from_numpy(b.k_pool.reshape(b.num_blocks, -1).view(np.uint8)[ids]).to(dev)
        assert torch.equal(reps[-1].k_pool.view(b.num_blocks, -1).view(torch.uint8)[ids_d.long()], ref_k), \
            "prefix restore mismatch"
        import_bytes = (len(imp[0]) and sum(2 * t[2] for t in imp[0])) * len(ids) + 4 * len(ids)

    def step(k, evs, split):
        """One step: restore replica k % R's prefix, then attend over replica
        (k+1) % R.  split=False times the whole attention call with one event
        pair; split=True records an event between its two kernels as well."""
        r_imp, r_att = k % R, (k + 1) % R
        evs[0].record(stream)
        if imp is not None:
            sg.specgen_kv_import(imp[r_imp], ids_d, b.num_blocks, stream=stream)
        evs[1].record(stream)
        if q_len is not None:   # one entry point, no separate phases
            sg.specgen_fork_prefill_attn(reps[r_att], q_len, out, lse, ws, stream=stream)
            evs[2].record(stream)
        elif split:
            sg.specgen_fork_decode_attn_phase(reps[r_att], sg.SPECGEN_PHASE_PARTIALS, None, None, ws, stream=stream)
            evs[2].record(stream)
            sg.specgen_fork_decode_attn_phase(reps[r_att], sg.SPECGEN_PHASE_MERGE, out, lse, ws, stream=stream)
        else:
            sg.specgen_fork_decode_attn(reps[r_att], out, lse, ws, stream=stream)
        evs[3].record(stream)

    if args.timeline:
        timeline_report(args, b, step, q_len)
        return
    total = args.warmup + args.steps
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(total)]
    log(f"warmup {args.warmup}")
    for k in range(args.warmup):
        step(k, events[k], False)
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    # A GPU-side spin (~20 ms) ahead of the timed steps lets the host queue all
    # of them before the GPU reaches the first, so the events measure GPU
    # execution only, not gaps where the GPU waits for the next launch.
    torch.cuda._sleep(SPIN_CYCLES)
    t0 = time.perf_counter()
    for k in range(args.warmup, total):
        step(k, events[k], False)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # GPU time of the timed steps (import + attention each), first event to last
    step_ms = events[args.warmup][0].elapsed_time(events[total - 1][3]) / args.steps
    timed = events[args.warmup:]
    imp_ms = np.array([e[0].elapsed_time(e[1]) for e in timed])
    attn_ms = np.array([e[1].elapsed_time(e[3]) for e in timed])
    # the same steps again with an event between the two kernels: the partial
    # kernel's own duration (the roofline figure) and the merge's
    log(f"timing {args.steps} steps with the phases split" if q_len is None else f"timing {args.steps} more steps")
    sevents = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda._sleep(SPIN_CYCLES)
    for k in range(args.steps):
        step(total + k, sevents[k], True)
    torch.cuda.synchronize()
    part_ms = np.array([e[1].elapsed_time(e[2]) for e in sevents])
    merge_ms = np.array([e[2].elapsed_time(e[3]) for e in sevents])
    # The partial kernel's average launch duration (the roofline figure):
    # `steps` launches back to back between one event pair, the replicas in
    # rotation (cold).  An event right before a launch delays the kernel's
    # start by several microseconds of dispatch, which the per-step split
    # above includes; back to back the launches follow each other as the
    # kernel trace shows them.
    b2b_ms = None
    if q_len is None:
        log(f"timing {args.steps} partial-kernel launches back to back")
        for k in range(R):
            sg.specgen_fork_decode_attn_phase(reps[k], sg.SPECGEN_PHASE_PARTIALS, None, None, ws, stream=stream)
        bev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        torch.cuda._sleep(SPIN_CYCLES)
        bev[0].record(stream)
        for k in range(args.steps):
            sg.specgen_fork_decode_attn_phase(reps[(k + 1) % R], sg.SPECGEN_PHASE_PARTIALS, None, None, ws,
                                              stream=stream)
        bev[1].record(stream)
        torch.cuda.synchronize()
        b2b_ms = bev[0].elapsed_time(bev[1]) / args.steps
    # whole calls back to back the same way (no import or event between them)
    cev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    torch.cuda._sleep(SPIN_CYCLES)
    cev[0].record(stream)
    for k in range(args.steps):
        if q_len is not None:
            sg.specgen_fork_prefill_attn(reps[(k + 1) % R], q_len, out, lse, ws, stream=stream)
        else:
            sg.specgen_fork_decode_attn(reps[(k + 1) % R], out, lse, ws, stream=stream)
    cev[1].record(stream)
    torch.cuda.synchronize()
    calls_b2b_ms = cev[0].elapsed_time(cev[1]) / args.steps

    def call(fb, st):   # the attention call alone
        if q_len is not None:
            sg.specgen_fork_prefill_attn(fb, q_len, out, lse, ws, stream=st)
        else:
            sg.specgen_fork_decode_attn(fb, out, lse, ws, stream=st)

    def pairs(n):
        return [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(n)]

    # warm: the call repeated on one replica, whose data the caches keep as far
    # as they hold it (172 MB of the 32k-prefix step fits the 256 MB MALL)
    log(f"timing {args.steps} warm calls")
    for _ in range(3):
        call(reps[1], stream)
    wev = pairs(args.steps)
    torch.cuda.synchronize()
    torch.cuda._sleep(SPIN_CYCLES)
    for k in range(args.steps):
        wev[k][0].record(stream)
        call(reps[1], stream)
        wev[k][1].record(stream)
    torch.cuda.synchronize()
    warm_ms = np.array([e[0].elapsed_time(e[1]) for e in wev])
    # HIP graphs: one captured call per replica, replayed in rotation (cold, like
    # the eager steps; no host work between the kernels of a call)
    log(f"timing {args.steps} graph replays")
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    graphs = []
    with torch.cuda.stream(side):
        for fb in reps:   # library and module set-up outside the capture
            call(fb, side)
    for fb in reps:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            call(fb, side)
        graphs.append(g)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    gev = pairs(args.steps)
    for k in range(R):
        graphs[k].replay()
    torch.cuda.synchronize()
    torch.cuda._sleep(SPIN_CYCLES)
    for k in range(args.steps):
        gev[k][0].record(stream)
        graphs[(k + 1) % R].replay()
        gev[k][1].record(stream)
    torch.cuda.synchronize()
    graph_ms = np.array([e[0].elapsed_time(e[1]) for e in gev])
    del graphs
    # the steps on either side of the restore, each timed on its own: export
    # (the prefix blocks migrate out to staging, the reverse of the import)
    # and append (every fork's next token written into its suffix blocks at
    # slot S_f, a fresh block where S_f is a multiple of 16; the suffix
    # lengths the attention reads are unchanged, so its inputs stay valid)
    moves = {}
    if imp is not None:
        log(f"timing {args.steps} exports")
        exp = [[(st, pl, bb_) for (pl, st, bb_) in tensors] for tensors in imp]
        xevents = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        torch.cuda._sleep(SPIN_CYCLES)
        for k in range(args.steps):
            xevents[k][0].record(stream)
            sg.specgen_kv_export(exp[k % R], ids_d, b.num_blocks, stream=stream)
            xevents[k][1].record(stream)
        torch.cuda.synchronize()
        assert torch.equal(imp[0][0][1], torch.from_numpy(ks.reshape(-1).view(np.uint8)).to(dev)), "export mismatch"
        exp_ms = np.array([e[0].elapsed_time(e[1]) for e in xevents])
        moves["export"] = {"blocks": int(len(ids)), "bytes": int(import_bytes),
                           "us": round(float(exp_ms.mean()) * 1e3, 2),
                           "gbps": round(import_bytes / (float(exp_ms.mean()) / 1e3) / 1e9, 2)}
    try:
        app = synth.make_append_case(b, seed=1)
    except AssertionError:      # the pool has no free block for a fork at a block boundary
        app = None
    if app is not None:
        log(f"timing {args.steps} appends")
        el = torch.uint8 if b.kv_dtype != "bf16" else torch.int16
        kvdt = sg.SPECGEN_FP8_E4M3 if b.kv_dtype != "bf16" else sg.SPECGEN_BF16
        a_dev = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in
                 (app.k_new, app.v_new, app.pos, app.suffix_table_off, app.suffix_table)]
        a_dev[0], a_dev[1] = a_dev[0].view(el), a_dev[1].view(el)
        aevents = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        torch.cuda._sleep(SPIN_CYCLES)
        for k in range(args.steps):
            fb = reps[k % R]
            aevents[k][0].record(stream)
            sg.specgen_kv_append(fb.k_pool, fb.v_pool, *a_dev, b.num_kv_heads, D, kv_dtype=kvdt,
                                 num_blocks=b.num_blocks, stream=stream)
            aevents[k][1].record(stream)
        torch.cuda.synchronize()
        app_ms = np.array([e[0].elapsed_time(e[1]) for e in aevents])
        app_bytes = app.algorithmic_bytes()
        moves["append"] = {"forks": N, "fresh_blocks": int(app.fresh_blocks.size), "bytes": int(app_bytes),
                           "us": round(float(app_ms.mean()) * 1e3, 2),
                           "gbps": round(app_bytes / (float(app_ms.mean()) / 1e3) / 1e9, 2)}
    attn_bytes = b.algorithmic_bytes() + (Q - N) * Hq * (D * 2 * 2 + 4)   # extra queries: q in, out and lse out
    out_bytes = Q * Hq * (D * 2 + 4)
    kern_bytes = attn_bytes - out_bytes      # the partial kernel reads everything but writes no output
    attn_s = float(np.median(attn_ms)) / 1e3
    part_s = (b2b_ms if b2b_ms is not None else float(np.median(part_ms))) / 1e3
    value = attn_bytes / attn_s / 1e9
    achieved = kern_bytes / part_s / 1e9
    # matrix work of the partial kernel: S = q K^T and P V over every key of
    # every (fork, q head) row, 2 flops per multiply-add each
    keys = sum(b.keys_of_fork(f) for f in range(N))   # prefix chain + suffix of every fork
    if q_len is not None:   # query i of fork f sees its suffix up to its own position
        keys = sum(int(q_len[f]) * b.keys_of_fork(f) - sum(int(q_len[f]) - 1 - i for i in range(int(q_len[f])))
                   for f in range(N))
    kern_flops = 4.0 * D * Hq * keys
    fp8 = b.kv_dtype != "bf16"
    if fp8 or q_len is not None:   # E4M3 KV (2r/e flop per byte) or many query rows: above the MFMA ridge
        tflops = kern_flops / part_s / 1e12
        kname = partial_kernel(D, fp8, args.fp8_scores) + (" (partials phase)" if q_len is None else
                                          " + merge (the whole prefill call: no separate phases)")
        roofline = {"kernel": kname, "bound": "mfma",
                    "achieved": round(tflops, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": traffic_from_profile(args.workload + ("_fp8scores" if args.fp8_scores else "")),
                    "algorithmic_flops_per_launch": int(kern_flops), "hbm_gbps": round(achieved, 2),
                    "launch_us": round(part_s * 1e6, 2)}
    else:
        roofline = {"kernel": partial_kernel(D, False, False) + " (partials phase)", "bound": "hbm",
                    "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic_from_profile(args.workload + ("_fp8scores" if args.fp8_scores else "")),
                    "algorithmic_bytes_per_launch": int(kern_bytes), "launch_us": round(part_s * 1e6, 2)}
    res = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(step_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "traces": b.num_traces, "forks": N,
                   "prefix_len": [int(x) for x in b.prefix_len[:4]], "suffix_tokens": int(b.suffix_len.sum()),
                   "q_heads": Hq, "kv_heads": b.num_kv_heads, "head_dim": D, "kv_dtype": b.kv_dtype,
                   "path": args.path, "fp8_scores": bool(args.fp8_scores), "replicas": R, "prefill_queries_per_fork": prefill_q or 0, "import_blocks": int(len(ids)) if imp is not None else 0},
        "pct_of_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "fork_tokens_per_s": round(Q / attn_s, 1),
        "gbps_back_to_back": round(attn_bytes / (calls_b2b_ms / 1e3) / 1e9, 2),
        "attn_us": {"p50": pct(attn_ms, 50), "p10": pct(attn_ms, 10), "p90": pct(attn_ms, 90),
                    "mean": round(float(attn_ms.mean()) * 1e3, 2),
                    "partials_p50": pct(part_ms, 50), "merge_p50": pct(merge_ms, 50),
                    "partials_back_to_back": round(b2b_ms * 1e3, 2) if b2b_ms is not None else None,
                    "calls_back_to_back": round(calls_b2b_ms * 1e3, 2),
                    "warm_p50": pct(warm_ms, 50), "graph_p50": pct(graph_ms, 50), "graph_p10": pct(graph_ms, 10),
                    "graph_p90": pct(graph_ms, 90),
                    "note": "whole call between two events, cold (value uses p50); partials/merge: the kernels "
                            "timed separately in a second run of the same steps (an event before each kernel); "
                            "partials_back_to_back: the partial kernel's mean launch duration over `steps` "
                            "launches between one event pair, replicas in rotation (the roofline figure); "
                            "calls_back_to_back: the whole call the same way; warm: "
                            "the call repeated on one replica; graph: one captured call per replica replayed in "
                            "rotation (cold)"},
        "attn_algorithmic_bytes": int(attn_bytes),
        "roofline": roofline,
    }
    if imp is not None:
        res["import"] = {"blocks": int(len(ids)), "bytes": int(import_bytes), "us": round(float(imp_ms.mean()) * 1e3, 2),
                         "gbps": round(import_bytes / (float(imp_ms.mean()) / 1e3) / 1e9, 2)}
    res.update(moves)
    log("streaming ceilings")
    res["stream_ceiling"] = stream_ceilings(dev, stream, batch=b, fb=reps)
    res["stream_ceiling"]["attn_frac_of_read"] = round(value / res["stream_ceiling"]["read_gbps"], 4)
    if roofline["bound"] == "hbm":
        res["stream_ceiling"]["partials_frac_of_slice_ring"] = round(
            achieved / res["stream_ceiling"]["slice_ring_gbps"], 4)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        res["cpu_baseline"] = cpu_baseline(b, args.cpu_seconds, q_len, attn_bytes)
        cb = res["cpu_baseline"]
        if cb["value"] > 0:   # the GPU call's rate over the oracle's, both on this machine and in the same unit
            cb["gpu_over_oracle"] = round(value / cb["value"], 1)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
