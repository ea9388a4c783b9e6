"""Decision-step throughput of the LayerCheck HIP library on one MI355X.

One step = one pass of the whole hot path over one synthetic model state
already resident in HBM: score every layer (segmented reduction over the live
weights and the shadow), select (threshold + staleness guard) and pack the
selected layers' weights, fp32 master copy and Adam m/v into one staging
buffer.  Between steps a synthetic optimizer update (not timed) produces the
next state.  The default workload is the Llama-3-8B-shaped state (bf16
weights + fp32 master + fp32 m/v + bf16 shadow, 8.03 B parameters, 35 layer
groups, S_max = 8, threshold calibrated to select about 20% of the layers per
step).

Timing: each decision step is bracketed by a device synchronise, and HIP
events on the library's stream time the step and each call; the reported
value is algorithmic bytes / GPU time.  The CPU baseline times the oracle
(score + select + pack of one transformer block) on the host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
CHUNK_BYTES = int(os.environ.get("LC_CHUNK_BYTES", 8 * 1024))  # score chunk (bytes of W per partial)
METRIC = "GB/s of model state scored+packed per decision step (% of HBM peak); ms/step"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed decision steps (default 2*S_max)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed decision steps (default S_max)")
    ap.add_argument("--workload", default=None,
                    help="default: llama3-8b; llama3.2-1b for --store-bench and --restore-bench")
    ap.add_argument("--mode", choices=["accum", "snapshot"], default="accum")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 4 GiB device copy (counter calibration)")
    ap.add_argument("--adamw", action="store_true",
                    help="drive the state with the fused AdamW + drift step instead of the standalone score")
    ap.add_argument("--sgd", action="store_true",
                    help="drive the state with the fused SGD + drift step (weights-only records)")
    ap.add_argument("--ceilings", action="store_true",
                    help="run the HBM ceiling probe (read, copy, 2-read-1-write streams with the kernels' "
                         "tile and block mapping) and print its JSON line")
    ap.add_argument("--torch-adamw-reference", action="store_true",
                    help="with --adamw: also time torch's fused AdamW (no drift) on the same parameter "
                         "shapes, plus the bf16 weight copy, as a reference point")
    ap.add_argument("--store-bench", default=None, metavar="DIR",
                    help="measure draining packed records into a persistence store in DIR and restoring "
                         "from it (default workload llama3.2-1b)")
    ap.add_argument("--restore-bench", action="store_true",
                    help="measure the composite restore from device-resident and from pinned-host versions "
                         "(default workload llama3.2-1b)")
    ap.add_argument("--no-placement-ceiling", action="store_true",
                    help="skip timing the score and copy access patterns with no arithmetic over the same arrays "
                         "after the timed steps (the ceiling of this placement in the memory interleave)")
    ap.add_argument("--placement-ceiling", action="store_true",
                    help="(the default) time those patterns after the timed steps")
    ap.add_argument("--placement-sweep", action="store_true",
                    help="also time the score pattern over the same arrays shifted "
                         "against each other by a set of byte offsets, and the copy into the staging buffer at "
                         "a set of offsets")
    ap.add_argument("--k0", type=float, default=None,
                    help="base threshold (skips the calibration window)")
    ap.add_argument("--json-out", default=None)
    return ap.parse_args()


# The sources each profiled kernel is compiled from: counter files taken on
# other sources are not reported.
KERNEL_SOURCES = {
    "score_kernel": ("lc_device.h", "lc_internal.h", "lc_kernels.hip"),
    "adamw_kernel": ("lc_device.h", "lc_internal.h", "lc_optim.hip"),
    "sgd_kernel": ("lc_device.h", "lc_internal.h", "lc_optim.hip"),
}


def kernel_source_hash(kernel: str = "score_kernel") -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, "paper_2609_27193_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str, mode: str):
    """HBM bytes per launch of ``kernel`` from committed rocprofv3 counter
    runs, only if they were taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_{mode}_pmc.json")
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    if d.get("kernel_source_hash") != kernel_source_hash(kernel):
        return None
    return d.get("hbm_bytes_per_launch")


def stream_hold(stream, us: float = 1000.0):
    """Returns a function that enqueues a spin kernel of about `us` microseconds
    on `stream` (torch's sleep kernel, its cycle count calibrated here once).
    Enqueued right before a step's first timing event, it keeps the stream busy
    while the host issues the step's calls, so the event fires when the GPU
    reaches the step rather than when the host does: the timed region then
    holds the step's GPU work and its own host round trips, not the host's
    latency in issuing the first call."""
    import torch
    if not hasattr(torch.cuda, "_sleep"):
        log("[bench] this torch has no sleep kernel: steps are timed without holding the stream")
        return lambda: None
    cycles = 1 << 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(cycles)  # first launch: compile / load
    e0.record(stream)
    torch.cuda._sleep(cycles)
    e1.record(stream)
    torch.cuda.synchronize()
    per_us = cycles / max(e0.elapsed_time(e1) * 1e3, 1e-3)
    n = max(1, int(per_us * us))
    return lambda: torch.cuda._sleep(n)


def copy_calibration(dev):
    """One plain 4 GiB device-to-device copy, for scaling the HBM byte
    counters of a profiling run."""
    import torch
    a_ = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    b_ = torch.empty_like(a_)
    a_.fill_(1.0)
    b_.copy_(a_)
    torch.cuda.synchronize()
    del a_, b_


def calibrate_k0(u_hist: np.ndarray, embed_mask: np.ndarray, s_max: int, target: float) -> float:
    """Base threshold K0 (embeddings get 10x) whose decision rule selects
    ``target`` of the layers per step on average, replaying the observed
    per-step scores (in ACCUM mode they do not depend on the selection)."""
    T, N = u_hist.shape
    horizon = max(8 * s_max, 4 * T)
    mult = np.where(embed_mask, 10.0, 1.0)

    def frac(k0):
        K = k0 * mult
        delta = np.zeros(N)
        last = np.zeros(N, dtype=np.int64)
        tot = 0
        for t in range(1, horizon + 1):
            delta += u_hist[(t - 1) % T]
            sel = (delta >= K) | (t - last >= s_max)
            delta[sel] = 0.0
            last[sel] = t
            tot += int(sel.sum())
        return tot / (horizon * N)

    lo, hi = -8.0, 2.0
    for _ in range(40):
        mid = 0.5 * (lo + hi)
        if frac(10.0 ** mid) > target:
            lo = mid
        else:
            hi = mid
    return 10.0 ** hi


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_baseline(state, spec, mode_name, sel_fraction, n_blocks=16):
    """Time the oracle (unchanged, numpy fp64) on a bounded sample of the same
    state with the GPU step's mix: ``n_blocks`` transformer blocks, of which
    the share of parameters the timed GPU steps selected on average is
    selected (K0 = 0 for those blocks, no threshold the others can reach, no
    staleness due) and packed; host copies made beforehand, not timed.  The
    oracle holds one layer per instance, so the sample runs as one instance
    per block: first one after the other on one thread, then spread over a
    thread per visible core (numpy releases the interpreter lock in its array
    loops)."""
    from concurrent.futures import ThreadPoolExecutor
    from oracle import layercheck_oracle as O
    from paper_2609_27193_amd.inputs import to_numpy_weight

    blocks = [i for i, l in enumerate(spec.layers) if l.name.startswith("block_")][:n_blocks]
    k_sel = max(1, int(round(sel_fraction * len(blocks))))
    dt = O.DT_BF16 if spec.weight_dtype == "bf16" else O.DT_F32
    mode = O.MODE_ACCUM if mode_name == "accum" else O.MODE_SNAPSHOT
    w = spec.weight_bytes
    t0 = time.perf_counter()
    host = []
    for b in blocks:
        segs = [s for s in state.segments if s.layer == b]
        a, e = segs[0].offset, segs[-1].offset + segs[-1].numel
        arrs = {"W": to_numpy_weight(state.weight[a:e]), "S": to_numpy_weight(state.shadow[a:e]),
                "M": None if state.master is None else state.master[a:e].cpu().numpy(),
                "m": state.exp_avg[a:e].cpu().numpy(), "v": state.exp_avg_sq[a:e].cpu().numpy()}
        host.append(([(s.offset - a, s.numel) for s in segs], arrs))
    copy_s = time.perf_counter() - t0
    n = sum(arrs["W"].size for _, arrs in host)
    n_sel = sum(host[i][1]["W"].size for i in range(k_sel))

    def make(i):
        cuts, arrs = host[i]
        osegs = [O.OSegment(0, arrs["W"][x:x + m], arrs["S"][x:x + m].copy(),
                            None if arrs["M"] is None else arrs["M"][x:x + m], arrs["m"][x:x + m],
                            arrs["v"][x:x + m]) for x, m in cuts]
        orc = O.LayerCheckOracle(osegs, 1, dt, spec.has_master, mode, [0.0 if i < k_sel else float("inf")],
                                 1 << 40)
        for (x, m), sg in zip(cuts, osegs):  # construction set S <- W: put the device shadow back
            sg.shadow[...] = arrs["S"][x:x + m]
        if mode == O.MODE_SNAPSHOT:
            orc.pack(0, 1 << 62)  # SNAPSHOT scores only after the pending base is packed (untimed)
        return orc

    def decide(orc):
        orc.score(1)
        mask, _ = orc.select(1, 1.0)
        payload, _ = orc.pack(0, 1 << 62)
        return int(mask[0]), len(payload)

    legs = []
    for threads in (1, max(1, min(len(blocks), len(os.sched_getaffinity(0))))):
        oracles = [make(i) for i in range(len(blocks))]
        t1 = time.perf_counter()
        if threads == 1:
            res = [decide(o) for o in oracles]
        else:
            with ThreadPoolExecutor(threads) as pool:
                res = list(pool.map(decide, oracles))
        elapsed = time.perf_counter() - t1
        assert [r[0] for r in res] == [int(i < k_sel) for i in range(len(blocks))]
        payload = sum(r[1] for r in res)
        score_bytes = (3 if mode == O.MODE_ACCUM else 2) * w * n
        pack_bytes = n_sel * (w + 4 * (3 if spec.has_master else 2)) + payload + (w * n_sel if mode == O.MODE_SNAPSHOT else 0)
        legs.append({"value": round((score_bytes + pack_bytes) / elapsed / 1e9, 4), "cores": threads,
                     "seconds": round(elapsed, 2)})
        del oracles
    best = legs[-1]
    return {"value": best["value"], "unit": "GB/s", "cores": best["cores"], "kind": "oracle",
            "legs": legs,
            "sample": f"{len(blocks)} transformer blocks ({n} params) of the same state after one more "
                      f"synthetic step; score all, select and pack {k_sel} ({n_sel / n:.1%} of the params, "
                      f"the timed steps selected {sel_fraction:.1%}); host copy {copy_s:.1f} s excluded; "
                      f"numpy fp64, one oracle per block, {legs[0]['seconds']:.1f} s on 1 thread, "
                      f"{best['seconds']:.1f} s on {best['cores']} threads; {cpu_model()}, "
                      f"{len(os.sched_getaffinity(0))} cores visible"}


# Blocks per CU at which the probe times each pattern (0: as many as fit).
PROBE_BLOCKS_PER_CU = (0, 2, 3, 4, 6)


def placement_ceiling(state, staging, mode_name, score_gbs, pack_gbs, sweep=False):
    """The access patterns of the score and pack kernels with no arithmetic
    (the kernels' tile and block mapping, from the probe library) over the
    very arrays the timed steps used: ACCUM's two reads and one write over W
    and S (S <- W, which the last ACCUM score already left in place), or
    SNAPSHOT's two reads, and a copy from the largest fp32 array into the
    staging buffer.  A kernel's rate over this ceiling is what its arithmetic
    and tables cost on top of where the arrays sit in the memory interleave."""
    import ctypes as C
    import torch
    from paper_2609_27193_amd.build_lib import PROBE_LIB
    if not os.path.exists(PROBE_LIB):
        log("[bench] no probe library (built by __graft_entry__.build()): placement ceiling not measured")
        return None
    lib = C.CDLL(PROBE_LIB)
    lib.lc_probe_arrays.restype = C.c_int
    lib.lc_probe_arrays.argtypes = [C.c_int, C.c_void_p, C.c_void_p, C.c_uint64, C.c_int, C.c_int,
                                    C.POINTER(C.c_double)]
    torch.cuda.synchronize()

    def rate(pattern, a, b, nbytes, blocks_per_cu=0):
        g = C.c_double()
        if lib.lc_probe_arrays(pattern, a, b, nbytes, 8, blocks_per_cu, C.byref(g)) != 0:
            raise RuntimeError("lc_probe_arrays failed")
        return g.value

    def best(pattern, a, b, nbytes):
        """The pattern at each number of blocks per CU (0: as many as fit);
        the ceiling is the best of them."""
        by_k = {k: round(rate(pattern, a, b, nbytes, k), 1) for k in PROBE_BLOCKS_PER_CU}
        k = max(by_k, key=by_k.get)
        return by_k[k], k, by_k

    w_bytes = state.weight.numel() * state.weight.element_size()
    score_pattern = 3 if mode_name == "accum" else 1
    ceil_score, k_score, score_by_k = best(score_pattern, state.weight.data_ptr(), state.shadow.data_ptr(), w_bytes)
    src = state.master if state.master is not None else state.exp_avg
    n = min(src.numel() * 4, staging.numel())
    ceil_copy, k_copy, copy_by_k = best(2, src.data_ptr(), staging.data_ptr(), n)
    out = {"score_pattern": "r2w1" if score_pattern == 3 else "read2", "score_gbs": round(ceil_score, 1),
           "score_kernel_frac": round(float(score_gbs) / ceil_score, 4), "copy_gbs": round(ceil_copy, 1),
           "copy_bytes": n, "score_gbs_by_blocks_per_cu": score_by_k, "copy_gbs_by_blocks_per_cu": copy_by_k}
    if pack_gbs:
        out["pack_kernel_frac"] = round(float(pack_gbs) / ceil_copy, 4)
    if sweep:
        # the shadow (or both arrays) entered `off` bytes later: tiles then pair
        # W and S at other relative positions of the interleave
        # (each at the number of blocks per CU that gave the ceiling above)
        offs = (0, 256, 1024, 4096, 8192, 20480, 65536, 1 << 20)
        out["score_vs_shadow_offset"] = {
            o: round(rate(score_pattern, state.weight.data_ptr(), state.shadow.data_ptr() + o, w_bytes - (1 << 20),
                          k_score), 1)
            for o in offs}
        out["score_vs_both_offset"] = {
            o: round(rate(score_pattern, state.weight.data_ptr() + o, state.shadow.data_ptr() + o, w_bytes - (1 << 20),
                          k_score), 1)
            for o in offs}
        out["copy_vs_staging_offset"] = {
            o: round(rate(2, src.data_ptr(), staging.data_ptr() + o, n - (1 << 20), k_copy), 1) for o in offs}
        if score_pattern == 3:  # the shifted r2w1 runs wrote W's bytes into S at an offset: S <- W again
            state.shadow.copy_(state.weight)
            torch.cuda.synchronize()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark measures one GPU only; --gpus must be 1 "
                                   "(the decision step is per-rank: each rank would run it on its own shard)"}))
        sys.exit(2)
    if args.ceilings:
        # a child process of its own: this process has not touched the GPU yet
        from paper_2609_27193_amd.build_lib import HBM_PROBE
        if not os.path.exists(HBM_PROBE):
            raise SystemExit("the HBM probe is built by __graft_entry__.build()")
        r = subprocess.run([HBM_PROBE], capture_output=True, text=True, timeout=600)
        if r.returncode != 0:
            raise SystemExit(r.stderr)
        print(r.stdout.strip(), flush=True)
        return
    import torch
    from paper_2609_27193_amd import inputs as I
    from paper_2609_27193_amd import layercheck as LC

    if args.workload is None:
        args.workload = "llama3.2-1b" if (args.store_bench or args.restore_bench) else "llama3-8b"
    if args.store_bench:
        return main_store(args, I.WORKLOADS[args.workload]())
    if args.restore_bench:
        return main_restore(args, I.WORKLOADS[args.workload]())
    spec = I.WORKLOADS[args.workload]()
    if args.adamw or args.sgd:
        return main_optim(args, spec, "sgd" if args.sgd else "adamw")
    s_max = spec.s_max
    steps = args.steps if args.steps is not None else 2 * s_max
    warmup = args.warmup if args.warmup is not None else s_max
    mode = LC.LC_MODE_ACCUM if args.mode == "accum" else LC.LC_MODE_SNAPSHOT
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    LC.load_library()

    t0 = time.perf_counter()
    log(f"[bench] {spec.name}: {spec.numel} params, {spec.n_layers} layers, mode {args.mode}")
    state = I.SyntheticState(spec, device=dev)
    torch.cuda.synchronize()
    log(f"[bench] state {state.nbytes() / 1e9:.2f} GB generated in {time.perf_counter() - t0:.1f} s")
    segs = LC.segments_from_state(state)
    dtype = LC.LC_DT_BF16 if spec.weight_dtype == "bf16" else LC.LC_DT_F32
    embed = np.array([l.name == "embed_tokens" for l in spec.layers])

    # -- calibration: record the per-step scores over one staleness period ----
    t = 0
    if args.k0 is None:
        probe = LC.LayoutDesc(segs, spec.n_layers, dtype, spec.has_master, LC.LC_MODE_ACCUM,
                              [float("inf")] * spec.n_layers, s_max, stream=stream.cuda_stream)
        ctx = LC.lc_init_layout(probe)
        u_hist = []
        for _ in range(s_max):
            t += 1
            state.step(t)
            LC.lc_score_layers(ctx, t)
            LC.lc_select(ctx, t, 1.0)
            u_hist.append(LC.lc_read_state(ctx, spec.n_layers)[0])
        LC.lc_destroy(ctx)
        k0_base = calibrate_k0(np.array(u_hist), embed, s_max, spec.target_fraction)
        log(f"[bench] calibrated K0 = {k0_base:.4g} (embeddings x10) for ~{spec.target_fraction:.0%} of layers")
    else:
        k0_base = args.k0
    k0 = [k0_base * (10.0 if e else 1.0) for e in embed]

    layout = LC.LayoutDesc(segs, spec.n_layers, dtype, spec.has_master, mode, k0, s_max,
                           t_base=t, stream=stream.cuda_stream)
    numel, rec = LC.lc_query_layout(layout)
    free, _ = torch.cuda.mem_get_info()
    cap = min(sum(rec), free - (8 << 30))
    cap = cap // 256 * 256
    staging = torch.empty(cap, dtype=torch.uint8, device=dev)
    log(f"[bench] staging {cap / 1e9:.2f} GB (all-layer worst case {sum(rec) / 1e9:.2f} GB)")
    ctx = LC.lc_init_layout(layout)
    LC.lc_pack_selected(ctx, staging.data_ptr(), cap, 0)  # part of the base version (untimed)

    n_chunks = sum(math.ceil(s.numel * spec.weight_bytes / CHUNK_BYTES) for s in state.segments)
    w = spec.weight_bytes
    P = spec.numel
    score_bytes = (3 if mode == LC.LC_MODE_ACCUM else 2) * w * P + 32 * n_chunks
    opt_b = 4 * (3 if spec.has_master else 2)

    if args.copy_calibration:
        copy_calibration(dev)

    hold = stream_hold(stream)
    rows = []
    for i in range(warmup + steps):
        t += 1
        state.step(t)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        hold()
        h0 = time.perf_counter()
        ev[0].record(stream)
        LC.lc_score_layers(ctx, t)
        ev[1].record(stream)
        mask, st = LC.lc_select(ctx, t, 1.0, spec.n_layers)
        ev[2].record(stream)
        rank, packed = 0, 0
        while True:
            r = LC.lc_pack_selected(ctx, staging.data_ptr(), cap, rank)
            packed += r["bytes_written"]
            if r["done"]:
                break
            rank = r["next_rank"]
        ev[3].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - h0
        sel_elems = int(sum(numel[l] for l in range(spec.n_layers) if mask[l]))
        pack_bytes = sel_elems * (w + opt_b) + packed + (w * sel_elems if mode == LC.LC_MODE_SNAPSHOT else 0)
        row = {"t": t, "step_ms": ev[0].elapsed_time(ev[3]), "score_ms": ev[0].elapsed_time(ev[1]),
               "select_ms": ev[1].elapsed_time(ev[2]), "pack_ms": ev[2].elapsed_time(ev[3]),
               "wall_ms": wall * 1e3, "n_sel": st["n_selected"], "n_forced": st["n_forced"],
               "pack_bytes": pack_bytes, "bytes": score_bytes + pack_bytes, "payload": packed,
               "sel_elems": sel_elems}
        log(f"[bench] {'warm' if i < warmup else 'time'} t={t} sel {st['n_selected']:2d}/{spec.n_layers} "
            f"(forced {st['n_forced']}) step {row['step_ms']:.3f} ms score {row['score_ms']:.3f} "
            f"select {row['select_ms']:.3f} pack {row['pack_ms']:.3f} "
            f"-> {row['bytes'] / row['step_ms'] / 1e6:.1f} GB/s")
        if i >= warmup:
            rows.append(row)
    LC.lc_destroy(ctx)

    tot_bytes = sum(r["bytes"] for r in rows)
    tot_ms = sum(r["step_ms"] for r in rows)
    value = tot_bytes / tot_ms / 1e6
    score_ms = np.mean([r["score_ms"] for r in rows])
    achieved = score_bytes / score_ms / 1e6
    pack_rows = [r for r in rows if r["pack_bytes"]]
    pack_gbs = (sum(r["pack_bytes"] for r in pack_rows) / sum(r["pack_ms"] for r in pack_rows) / 1e6
                if pack_rows else None)
    traffic = measured_traffic("score_kernel", args.workload, args.mode)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(tot_ms / len(rows), 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 in, f32->f64 reduce", "data": "synthetic",
        "config": {"workload": f"{spec.name}-shaped state, decision step ({args.mode})",
                   "params": P, "layer_groups": spec.n_layers, "s_max": s_max,
                   "target_selected_fraction": spec.target_fraction,
                   "selected_fraction": round(float(np.mean([r["n_sel"] for r in rows])) / spec.n_layers, 4),
                   "k0_base": k0_base, "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
                   "score_gbs": round(achieved, 1), "pack_gbs": None if pack_gbs is None else round(pack_gbs, 1),
                   "bytes_per_step_gb": round(tot_bytes / len(rows) / 1e9, 3)},
        "roofline": {"bound": "hbm", "kernel": "score_kernel (+finalize)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic},
    }
    if not args.no_placement_ceiling:
        out["placement_ceiling"] = placement_ceiling(state, staging, args.mode, achieved, pack_gbs,
                                                     args.placement_sweep)
        log(f"[bench] placement ceiling {out['placement_ceiling']}")
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample of the state")
        state.step(t + 1)  # fresh drift against the current shadow (untimed)
        torch.cuda.synchronize()
        sel_params = float(np.mean([r["sel_elems"] for r in rows])) / P
        out["cpu_baseline"] = cpu_baseline(state, spec, args.mode, sel_params)
    line = json.dumps(out)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")


def main_store(args, spec):
    """Persistence path: drain the full base version (every layer) and the
    selections of a few decision steps from device staging into a store
    (pinned ring, writer threads, fsync), then restore the composite state
    from the store.  Per step it times how long the staging buffer is held
    (the device-to-host copies, against a plain pinned copy of the same size
    as the host-link ceiling) and how long until the version is durable.
    Rates are over the payload bytes; the restore reads files the same
    process wrote, so they may come from the page cache."""
    import shutil
    import torch
    from paper_2609_27193_amd import inputs as I
    from paper_2609_27193_amd import layercheck as LC

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    LC.load_library()
    state = I.SyntheticState(spec, device=dev)
    segs = LC.segments_from_state(state)
    dtype = LC.LC_DT_BF16 if spec.weight_dtype == "bf16" else LC.LC_DT_F32
    k0 = [(args.k0 or 0.03) * (10.0 if l.name == "embed_tokens" else 1.0) for l in spec.layers]
    layout = LC.LayoutDesc(segs, spec.n_layers, dtype, spec.has_master, LC.LC_MODE_ACCUM, k0, spec.s_max,
                           stream=stream.cuda_stream)
    numel, rec = LC.lc_query_layout(layout)
    total = sum(rec)
    staging = torch.empty(total, dtype=torch.uint8, device=dev)
    w, opt_b = spec.weight_bytes, 4 * (3 if spec.has_master else 2)

    def step_bytes(mask, packed):
        """Algorithmic bytes of one ACCUM decision step: score 3wP, then the
        selected state read and the records written."""
        return 3 * w * spec.numel + sum(n for n, m in zip(numel, mask) if m) * (w + opt_b) + packed
    ctx = LC.lc_init_layout(layout)
    ring = 4 << 30
    # host-link ceiling: one plain device-to-pinned copy of the ring's size
    pinned = torch.empty(ring, dtype=torch.uint8, pin_memory=True)
    for _ in range(2):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        pinned.copy_(staging[:ring], non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
    link_gbs = ring / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del pinned
    log(f"[bench] host link: device-to-pinned copy of {ring / 2**30:.0f} GiB at {link_gbs:.1f} GB/s")
    if os.path.exists(args.store_bench):
        shutil.rmtree(args.store_bench)
    store = LC.Store(args.store_bench, rec, buffer_bytes=ring)
    res = LC.lc_pack_selected(ctx, staging.data_ptr(), total, 0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    store.append(0, np.ones(spec.n_layers, np.uint8), staging.data_ptr(), res["bytes_written"], stream.cuda_stream)
    t_append = time.perf_counter() - t0
    store.sync()
    t_base = time.perf_counter() - t0
    log(f"[bench] base version {total / 1e9:.2f} GB: append returned after {t_append:.2f} s, durable after "
        f"{t_base:.2f} s -> {total / t_base / 1e9:.2f} GB/s")
    drained, release_s, durable_s, call_s = 0, 0.0, 0.0, 0.0
    alone_ms, alone_bytes = [], 0
    for t in range(1, 7):
        state.step(t)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        LC.lc_score_layers(ctx, t)
        mask, st = LC.lc_select(ctx, t, 1.0, spec.n_layers)
        r = LC.lc_pack_selected(ctx, staging.data_ptr(), total, 0)
        e1.record(stream)
        torch.cuda.synchronize()
        alone_ms.append(e0.elapsed_time(e1))
        alone_bytes += step_bytes(mask, r["bytes_written"])
        a = time.perf_counter()
        store.append(t, mask, staging.data_ptr(), r["bytes_written"], stream.cuda_stream)
        b = time.perf_counter()
        stream.synchronize()  # the staging buffer is free again
        c = time.perf_counter()
        store.sync()
        d = time.perf_counter()
        call_s += b - a
        release_s += c - a
        durable_s += d - a
        drained += r["bytes_written"]
        log(f"[bench] t={t}: {st['n_selected']} layers, {r['bytes_written'] / 1e9:.2f} GB: append {b - a:.3f} s, "
            f"staging free after {c - a:.3f} s, durable after {d - a:.3f} s")
    # Overlapped drain: two staging buffers and lc_store_append_async.  The
    # caller's stream waits only for the copies out of the buffer it is about
    # to pack again, so each decision step runs while the previous step's
    # payload is still being copied out; its GPU time is compared with the
    # same step above, where nothing was in flight.
    od = args.store_bench.rstrip("/") + "_overlapped"
    shutil.rmtree(od, ignore_errors=True)
    ostore = LC.Store(od, rec, buffer_bytes=ring)
    stagings = [staging, torch.empty(total, dtype=torch.uint8, device=dev)]
    reuse = [torch.cuda.Event() for _ in stagings]
    for ev in reuse:
        ev.record(stream)  # creates the underlying event
    o_bytes, o_step_bytes, overlap_ms, o_call_s, marks = 0, 0, [], 0.0, []
    a = time.perf_counter()
    for t in range(7, 13):
        state.step(t)
        k = t % 2
        stream.wait_event(reuse[k])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        LC.lc_score_layers(ctx, t)
        mask, st = LC.lc_select(ctx, t, 1.0, spec.n_layers)
        r = LC.lc_pack_selected(ctx, stagings[k].data_ptr(), total, 0)
        e1.record(stream)
        b = time.perf_counter()
        ostore.append_async(t, mask, stagings[k].data_ptr(), r["bytes_written"], stream.cuda_stream,
                            reuse[k].cuda_event)
        o_call_s += time.perf_counter() - b
        marks.append((e0, e1))
        o_bytes += r["bytes_written"]
        o_step_bytes += step_bytes(mask, r["bytes_written"])
    torch.cuda.synchronize()
    ostore.sync()
    o_total_s = time.perf_counter() - a
    overlap_ms = [x.elapsed_time(y) for x, y in marks]
    ostore.close()
    shutil.rmtree(od, ignore_errors=True)
    del stagings[1]
    alone_gbs = alone_bytes / sum(alone_ms) / 1e6
    overlap_gbs = o_step_bytes / sum(overlap_ms) / 1e6
    log(f"[bench] overlapped drain: decision steps at {overlap_gbs:.0f} GB/s with the previous payload in flight "
        f"vs {alone_gbs:.0f} GB/s alone ({np.mean(overlap_ms):.2f} / {np.mean(alone_ms):.2f} ms per step); "
        f"append calls {o_call_s:.3f} s in total; {o_bytes / 1e9:.2f} GB durable after {o_total_s:.2f} s")
    t_fail = 5
    stored_before = sum(e["payload_bytes"] for e in store.entries())
    a = time.perf_counter()
    removed = store.compact(t_fail)  # keep what recovery at t_fail or later can use
    compact_s = time.perf_counter() - a
    stored_after = sum(e["payload_bytes"] for e in store.entries())
    log(f"[bench] compaction at t_keep={t_fail}: {stored_before / 1e9:.2f} GB -> {stored_after / 1e9:.2f} GB "
        f"({removed} files removed) in {compact_s:.3f} s")
    # fail-stop: lose the live state, recover the composite from the store
    for tnsr in (state.weight, state.shadow, state.master, state.exp_avg, state.exp_avg_sq):
        if tnsr is not None:
            tnsr.zero_()
    torch.cuda.synchronize()
    a = time.perf_counter()
    chosen = store.restore(ctx, t_fail)
    restore_s = time.perf_counter() - a
    # again: the first restore's buffered reads left the records in the page
    # cache, so this one measures the pipeline against the host link
    a = time.perf_counter()
    store.restore(ctx, t_fail)
    restore_warm_s = time.perf_counter() - a
    store.close()
    LC.lc_destroy(ctx)
    out = {"metric": "persistence store: drain and composite-restore GB/s", "unit": "GB/s",
           "config": {"workload": f"{spec.name}-shaped state", "params": spec.numel, "layer_groups": spec.n_layers,
                      "record_set_gb": round(total / 1e9, 3), "ring_gib": ring >> 30},
           "host_link_gbs": round(link_gbs, 2),
           "drain_base_gbs": round(total / t_base / 1e9, 3),
           "steps_gb": round(drained / 1e9, 3),
           # what full checkpoints at the same six steps would have written (Table 1's comparison)
           "full_checkpoints_gb": round(6 * total / 1e9, 3),
           "steps_append_call_s": round(call_s, 3),
           "steps_staging_release_gbs": round(drained / release_s / 1e9, 2),
           "steps_durable_gbs": round(drained / durable_s / 1e9, 3),
           # the caller's stream held per step by the drain: the device-to-host copies
           # with lc_store_append, none with lc_store_append_async
           "steps_stream_held_ms": round(release_s / 6 * 1e3, 2),
           "decision_step_gbs_alone": round(alone_gbs, 1),
           "decision_step_gbs_overlapped": round(overlap_gbs, 1),
           "overlapped_append_call_s": round(o_call_s, 3),
           "overlapped_durable_gbs": round(o_bytes / o_total_s / 1e9, 3),
           "stored_gb_before_compact": round(stored_before / 1e9, 3),
           "stored_gb_after_compact": round(stored_after / 1e9, 3), "compact_s": round(compact_s, 3),
           "restore_gbs": round(total / restore_s / 1e9, 3), "restore_s": round(restore_s, 3),
           "restore_warm_gbs": round(total / restore_warm_s / 1e9, 3),
           "restored_timestamps": sorted(set(int(x) for x in chosen))}
    print(json.dumps(out), flush=True)
    shutil.rmtree(args.store_bench, ignore_errors=True)


def main_restore(args, spec):
    """Composite recovery (Section 3.5) from a history of versions: the base
    at step 0 and the selections of up to three following decision steps (as
    many as device memory holds).  Timed with every version resident in
    device memory (the unpack kernel, against the HBM roofline) and, when the
    record set fits in 48 GB, with every version in pinned host memory
    (per-block host-to-device copies, against a plain pinned copy as the
    host-link ceiling).  Bytes: each layer's record read once, its arrays and
    its shadow written once."""
    import torch
    from paper_2609_27193_amd import inputs as I
    from paper_2609_27193_amd import layercheck as LC

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    LC.load_library()
    state = I.SyntheticState(spec, device=dev)
    segs = LC.segments_from_state(state)
    dtype = LC.LC_DT_BF16 if spec.weight_dtype == "bf16" else LC.LC_DT_F32
    k0 = [(args.k0 or 0.03) * (10.0 if l.name == "embed_tokens" else 1.0) for l in spec.layers]
    layout = LC.LayoutDesc(segs, spec.n_layers, dtype, spec.has_master, LC.LC_MODE_ACCUM, k0, spec.s_max,
                           stream=stream.cuda_stream)
    numel, rec = LC.lc_query_layout(layout)
    ctx = LC.lc_init_layout(layout)
    versions = []

    def pack(t, mask):
        nbytes = int(sum(rec[l] for l in range(spec.n_layers) if mask[l]))
        buf = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
        r = LC.lc_pack_selected(ctx, buf.data_ptr(), nbytes, 0)
        assert r["done"] and r["bytes_written"] == nbytes
        versions.append((t, mask.copy(), buf, nbytes))

    pack(0, np.ones(spec.n_layers, np.uint8))
    t_fail = 0
    for t in range(1, 4):  # up to three selections after the base: a mixed-timestamp composite
        state.step(t)
        LC.lc_score_layers(ctx, t)
        mask, st = LC.lc_select(ctx, t, 1.0, spec.n_layers)
        if st["payload_bytes"] + (8 << 30) > torch.cuda.mem_get_info()[0]:
            log(f"[bench] step {t}: {st['payload_bytes'] / 1e9:.1f} GB does not fit beside the history; stop")
            break
        pack(t, mask)
        t_fail = t
    torch.cuda.synchronize()
    with_host = versions[0][3] <= (48 << 30)
    host = []
    if with_host:
        host = [(t, m, torch.empty(max(n, 1), dtype=torch.uint8, pin_memory=True), n) for t, m, _, n in versions]
        for (_, _, d, n), (_, _, h, _) in zip(versions, host):
            h[:n].copy_(d[:n])
        torch.cuda.synchronize()
    w = spec.weight_bytes
    opt_b = 4 * (3 if spec.has_master else 2)
    moved = sum(numel[l] * (w + opt_b) for l in range(spec.n_layers))
    alg_bytes = 2 * moved + w * spec.numel  # record read + arrays written + shadow written

    def timed(vs):
        best = None
        chosen = None
        for _ in range(3):
            torch.cuda.synchronize()
            a = time.perf_counter()
            # the call returns once the restore has completed on the device
            chosen = LC.lc_restore_composite(
                ctx, [{"step": t, "mask": m, "payload": b.data_ptr() if n else 0, "payload_bytes": n}
                      for t, m, b, n in vs], t_fail, spec.n_layers)
            wall = time.perf_counter() - a
            best = wall if best is None else min(best, wall)
        return best, chosen

    if args.copy_calibration:
        copy_calibration(dev)
    dev_s, chosen = timed(versions)
    if with_host:
        host_s, chosen_h = timed(host)
        assert chosen.tolist() == chosen_h.tolist()
    # ceilings: plain copies of 4 GiB (the second of two), device-to-device and pinned host-to-device
    n_c = min(versions[0][3], 4 << 30)
    dst = torch.empty(n_c, dtype=torch.uint8, device=dev)

    def copy_rate(src, nbytes_moved):
        for _ in range(2):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            dst.copy_(src, non_blocking=True)
            e1.record(stream)
            torch.cuda.synchronize()
        return nbytes_moved / (e0.elapsed_time(e1) * 1e-3) / 1e9

    d2d_gbs = copy_rate(versions[0][2][:n_c], 2 * n_c)
    h2d_gbs = copy_rate(host[0][2][:n_c], n_c) if with_host else None
    LC.lc_destroy(ctx)
    out = {"metric": "composite restore GB/s (records read + state and shadow written)", "unit": "GB/s",
           "config": {"workload": f"{spec.name}-shaped state", "params": spec.numel, "layer_groups": spec.n_layers,
                      "versions": len(versions), "t_fail": t_fail,
                      "restored_timestamps": sorted(set(int(x) for x in chosen)),
                      "record_set_gb": round(moved / 1e9, 3), "algorithmic_gb": round(alg_bytes / 1e9, 3)},
           "device_versions": {"s": round(dev_s, 5), "gbs": round(alg_bytes / dev_s / 1e9, 1),
                               "frac_of_hbm_peak": round(alg_bytes / dev_s / 1e9 / HBM_PEAK_GBS, 4),
                               "plain_d2d_copy_gbs": round(d2d_gbs, 1)},
           "pinned_host_versions": ({"s": round(host_s, 4), "record_gbs": round(moved / host_s / 1e9, 2),
                                     "plain_h2d_copy_gbs": round(h2d_gbs, 2)} if with_host else None)}
    line = json.dumps(out)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")


ADAMW = dict(lr=1e-5, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


SGD = dict(lr=1e-4, weight_decay=0.1)


def main_optim(args, spec, optimizer):
    """Optimizer-driven decision step: the fused optimizer + drift pass (one
    read and write of the optimizer state, no shadow), then select and pack.
    AdamW records hold W, master, m and v; SGD keeps no moments, so its
    records hold W and master only (Section 4.7).  The gradients of each step
    are generated untimed."""
    import torch
    from paper_2609_27193_amd import inputs as I
    from paper_2609_27193_amd import layercheck as LC

    if args.mode != "accum":
        raise SystemExit("the optimizer-driven step accumulates (ACCUM mode)")
    adamw = optimizer == "adamw"
    s_max = spec.s_max
    steps = args.steps if args.steps is not None else 2 * s_max
    warmup = args.warmup if args.warmup is not None else s_max
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    LC.load_library()
    state = I.SyntheticState(spec, device=dev, shadow=False)
    torch.cuda.synchronize()
    log(f"[bench] {spec.name} ({optimizer}-driven, no shadow): state {state.nbytes() / 1e9:.2f} GB")
    segs = LC.segments_from_state(state)
    if not adamw:  # weights-only layout: the moments are not part of the state
        segs = [LC.Segment(s.layer, s.numel, s.weight, None, s.master, None, None) for s in segs]
    dtype = LC.LC_DT_BF16 if spec.weight_dtype == "bf16" else LC.LC_DT_F32
    embed = np.array([l.name == "embed_tokens" for l in spec.layers])
    decay = state.decay_mask()
    adam_t = 0

    def grad_ptrs(g):
        """One device address per segment (the layout's order) into the flat gradient."""
        base, esz = g.data_ptr(), g.element_size()
        return [base + s.offset * esz for s in state.segments]

    def fused(ctx, t, ptrs):
        if adamw:
            LC.lc_adamw_step_score(ctx, t, ptrs, LC.LC_DT_BF16, ADAMW["lr"], ADAMW["beta1"], ADAMW["beta2"],
                                   ADAMW["eps"], ADAMW["weight_decay"], adam_t, decay)
        else:
            LC.lc_sgd_step_score(ctx, t, ptrs, LC.LC_DT_BF16, SGD["lr"], SGD["weight_decay"], decay)

    t = 0
    if args.k0 is None:
        probe = LC.LayoutDesc(segs, spec.n_layers, dtype, spec.has_master, LC.LC_MODE_ACCUM,
                              [float("inf")] * spec.n_layers, s_max, stream=stream.cuda_stream)
        ctx = LC.lc_init_layout(probe)
        u_hist = []
        for _ in range(s_max):
            t += 1
            adam_t += 1
            g = state.gradients(t)
            fused(ctx, t, grad_ptrs(g))
            LC.lc_select(ctx, t, 1.0)
            u_hist.append(LC.lc_read_state(ctx, spec.n_layers)[0])
            del g
        LC.lc_destroy(ctx)
        k0_base = calibrate_k0(np.array(u_hist), embed, s_max, spec.target_fraction)
        log(f"[bench] calibrated K0 = {k0_base:.4g} (embeddings x10)")
    else:
        k0_base = args.k0
    k0 = [k0_base * (10.0 if e else 1.0) for e in embed]
    layout = LC.LayoutDesc(segs, spec.n_layers, dtype, spec.has_master, LC.LC_MODE_ACCUM, k0, s_max,
                           t_base=t, stream=stream.cuda_stream)
    numel, rec = LC.lc_query_layout(layout)
    free, _ = torch.cuda.mem_get_info()
    cap = min(sum(rec), free - (spec.numel * 2 + (12 << 30))) // 256 * 256  # room for the gradients
    staging = torch.empty(cap, dtype=torch.uint8, device=dev)
    ctx = LC.lc_init_layout(layout)
    LC.lc_pack_selected(ctx, staging.data_ptr(), cap, 0)
    w, P = spec.weight_bytes, spec.numel
    n_chunks = sum(math.ceil(s.numel * w / CHUNK_BYTES) for s in state.segments)
    # grad (bf16) read, master (and m, v for AdamW) read+written, weights written
    # (and read when they are the parameters)
    moments_b = 16 if adamw else 0
    opt_bytes = P * (2 + (8 if spec.has_master else 0) + moments_b + (w if spec.has_master else 2 * w)) \
        + 32 * n_chunks
    opt_b = (4 if spec.has_master else 0) + (8 if adamw else 0)  # fp32 bytes per element in a record
    if args.copy_calibration:
        copy_calibration(dev)
    hold = stream_hold(stream)
    rows = []
    for i in range(warmup + steps):
        t += 1
        adam_t += 1
        g = state.gradients(t)
        ptrs = grad_ptrs(g)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        hold()
        ev[0].record(stream)
        fused(ctx, t, ptrs)
        ev[1].record(stream)
        mask, st = LC.lc_select(ctx, t, 1.0, spec.n_layers)
        ev[2].record(stream)
        rank, packed = 0, 0
        while True:
            r = LC.lc_pack_selected(ctx, staging.data_ptr(), cap, rank)
            packed += r["bytes_written"]
            if r["done"]:
                break
            rank = r["next_rank"]
        ev[3].record(stream)
        torch.cuda.synchronize()
        del g
        sel_elems = int(sum(numel[l] for l in range(spec.n_layers) if mask[l]))
        pack_bytes = sel_elems * (w + opt_b) + packed
        row = {"step_ms": ev[0].elapsed_time(ev[3]), "opt_ms": ev[0].elapsed_time(ev[1]),
               "pack_ms": ev[2].elapsed_time(ev[3]), "n_sel": st["n_selected"], "pack_bytes": pack_bytes,
               "bytes": opt_bytes + pack_bytes}
        log(f"[bench] {'warm' if i < warmup else 'time'} t={t} sel {st['n_selected']:2d}/{spec.n_layers} "
            f"step {row['step_ms']:.3f} ms ({optimizer}+drift {row['opt_ms']:.3f}, pack {row['pack_ms']:.3f}) "
            f"-> {row['bytes'] / row['step_ms'] / 1e6:.1f} GB/s")
        if i >= warmup:
            rows.append(row)
    LC.lc_destroy(ctx)
    tot_bytes = sum(r["bytes"] for r in rows)
    tot_ms = sum(r["step_ms"] for r in rows)
    opt_ms = float(np.mean([r["opt_ms"] for r in rows]))
    out = {
        "metric": "GB/s of optimizer state updated+scored and packed per training step (% of HBM peak); ms/step",
        "value": round(tot_bytes / tot_ms / 1e6, 2), "unit": "GB/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": round(tot_ms / len(rows), 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": f"bf16 grads, f32 {optimizer}, f64 reduce",
        "data": "synthetic",
        "config": {"workload": f"{spec.name}-shaped state, fused {optimizer} + drift, select, pack",
                   "params": P, "layer_groups": spec.n_layers, "s_max": s_max, optimizer: ADAMW if adamw else SGD,
                   "selected_fraction": round(float(np.mean([r["n_sel"] for r in rows])) / spec.n_layers, 4),
                   "k0_base": k0_base, "opt_bytes_per_step_gb": round(opt_bytes / 1e9, 3)},
        "roofline": {"bound": "hbm", "kernel": f"optim_kernel<{optimizer}> (+finalize)",
                     "achieved": round(opt_bytes / opt_ms / 1e6, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(opt_bytes / opt_ms / 1e6 / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(f"{optimizer}_kernel", args.workload, "accum")},
    }
    if args.torch_adamw_reference and adamw:
        del state, staging
        torch.cuda.empty_cache()
        out["torch_fused_adamw_reference"] = torch_adamw_reference(spec, dev)
    line = json.dumps(out)
    print(line, flush=True)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")


def torch_adamw_reference(spec, dev, steps=5):
    """torch.optim.AdamW(fused=True) over one fp32 master tensor per layer of
    the same shapes (fp32 gradients, as that optimizer requires the
    parameter's dtype), followed by the bf16 weight copy that the fused
    AdamW + drift kernel writes in the same pass.  No drift is computed."""
    import torch
    params, weights = [], []
    for layer in spec.layers:
        n = sum(t.numel for t in layer.tensors)
        p = torch.nn.Parameter(torch.randn(n, device=dev) * 0.02)
        p.grad = torch.randn(n, device=dev)
        params.append(p)
        weights.append(torch.empty(n, dtype=torch.bfloat16, device=dev))
    opt = torch.optim.AdamW(params, lr=ADAMW["lr"], betas=(ADAMW["beta1"], ADAMW["beta2"]), eps=ADAMW["eps"],
                            weight_decay=ADAMW["weight_decay"], fused=True)
    stream = torch.cuda.current_stream()
    times = []
    for i in range(steps + 2):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        torch.cuda.synchronize()
        e[0].record(stream)
        opt.step()
        e[1].record(stream)
        with torch.no_grad():
            for w, p in zip(weights, params):
                w.copy_(p)
        e[2].record(stream)
        torch.cuda.synchronize()
        if i >= 2:
            times.append((e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])))
    opt_ms = float(np.mean([a for a, _ in times]))
    copy_ms = float(np.mean([b for _, b in times]))
    P = spec.numel
    log(f"[bench] torch fused AdamW {opt_ms:.2f} ms + bf16 weight copy {copy_ms:.2f} ms")
    return {"adamw_ms": round(opt_ms, 3), "weight_copy_ms": round(copy_ms, 3),
            "total_ms": round(opt_ms + copy_ms, 3),
            "bytes_gb": round(P * (28 + 6) / 1e9, 2),
            "note": "fp32 params and grads (28 B/param) + bf16 weight copy (6 B/param); no drift statistic"}


if __name__ == "__main__":
    main()
