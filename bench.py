#!/usr/bin/env python3
"""Decode-step benchmark of the SANTA / S2ANTA HIP path on one MI355X.

Workload (default): Llama-3.1-8B attention layer at 32k context, batch 1 --
32 query heads, 8 KV heads, head_dim 128, bf16, n_k = 32768, sink + 32
planted heavy keys per KV head, stratified sampling with S = 256 (seeded
synthetic inputs, see workload/gen.py).  One "step" is one call of
santa_decode_stratified over the whole batch.

Protocol (the paper's decode microbenchmark, adapted): inputs are built and
uploaded before timing; W untimed warm-up steps; then K timed steps, each
preceded (outside the timed region) by an in-place update of a 1 GiB buffer
(the paper's cache-thrash step) and a read-only pass over a second 2 GiB
buffer, so that neither L2 nor the 256 MB Infinity Cache holds the KV cache and
no dirty flush lines are left to be written back during the timed call; HIP
events recorded on the library's stream around each call.  The exact dense
kernel of the same library is timed the same way on the same inputs.

value = algorithmic bytes / mean step time, where algorithmic bytes = all keys
+ the unique value rows the step gathers (counted from idx_out in an untimed
call) + q + out + uniforms.  `attainable_read` times the library's
streaming-read calibration kernel (santa_stream_read) over the same number of
bytes under the same protocol: the rate a plain read of those bytes reaches on
this device, and the step's kernel rate as a fraction of it.  Prints one JSON
line.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn µs/step + HBM GB/s (% of peak) at 32k ctx, vs dense decode"
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cfg", type=int, default=2, help="workload configuration (1..5)")
    ap.add_argument("--B", type=int, default=None)
    ap.add_argument("--S", type=int, default=None)
    ap.add_argument("--kind", default=None,
                    help="dense | systematic | stratified | iid | bernoulli | flash")
    ap.add_argument("--tile", type=int, default=256, help="flash: keys per tile")
    ap.add_argument("--S-tile", type=int, default=None,
                    help="flash: draws per tile (default: the budget rule S_tile ~ S / T)")
    ap.add_argument("--layout", default="nhd", choices=["nhd", "hnd"])
    ap.add_argument("--path", default="auto", choices=["auto", "one", "two", "multi", "rows"],
                    help="launch path (santa_set_options): by size, one persistent launch, "
                         "key stream + per-head value stage, or the multi-kernel variant")
    ap.add_argument("--splits", type=int, default=0, help="KV splits per row (0: by size)")
    ap.add_argument("--mode", type=int, default=None,
                    help="Bernoulli: 0 per-head ternary query, 1 mean group query")
    ap.add_argument("--B-draws", type=int, default=None, help="Bernoulli: draws per feature")
    ap.add_argument("--kv", default="bf16", choices=["bf16", "fp8"],
                    help="cache element type: the query's (bf16) or OCP FP8 E4M3 codes with "
                         "per-(batch, KV head) scales (queries and outputs stay bf16)")
    ap.add_argument("--flush-gib", type=float, default=1.0)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--append", action="store_true",
                    help="pass the current token's rows as k_new / v_new: every call (sampled "
                         "and dense) writes them into the cache inside its launch")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--profile", action="store_true",
                    help="timed loops only (for rocprofv3 runs); still prints the JSON line")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        sys.stderr.write("bench.py: this build runs on exactly one GPU; --gpus N > 1 is not "
                         "supported (the decode step has no multi-GPU path here).\n")
        sys.exit(2)

    import torch
    from paper_2605_01910_amd import santa as S
    from workload import make_workload

    S.load()  # fails loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    over = {}
    if args.B is not None:
        over["B"] = args.B
    if args.S is not None:
        over["S"] = args.S
    if args.kind is not None:
        over["kind"] = args.kind
    if args.mode is not None:
        over["mode"] = args.mode
    if args.B_draws is not None:
        over["B_draws"] = args.B_draws
    if args.kv == "fp8":
        over["kv_dtype"] = "fp8"
    if args.kind == "flash":
        from workload.gen import CONFIGS
        n = CONFIGS[args.cfg]["n"]
        over["tile"] = args.tile
        over["S_tile"] = args.S_tile or flash_tile_budget(over.get("S", CONFIGS[args.cfg]["S"]),
                                                          (n + args.tile - 1) // args.tile)
    S.santa_set_options(S.PATHS[args.path], args.splits)
    t0 = time.time()
    w = make_workload(args.cfg, seed=0, **over)
    print(f"[bench] workload cfg={args.cfg} B={w.B} Hq={w.Hq} Hkv={w.Hkv} n={w.n_max} "
          f"kind={w.kind} S={w.S} built in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    from workload.device import DeviceWorkload, current_rows
    KIND_CODE = {"dense": S.SANTA_KIND_DENSE, "systematic": S.SANTA_KIND_SYSTEMATIC,
                 "stratified": S.SANTA_KIND_STRATIFIED, "bernoulli": S.SANTA_KIND_BERNOULLI,
                 "flash": S.SANTA_KIND_FLASH, "iid": S.SANTA_KIND_IID}
    dw = DeviceWorkload(w, layout=args.layout)
    kind = w.kind
    if args.append:
        if kind == "bernoulli":
            sys.exit("--append is not available with Bernoulli scores")
        rows = current_rows(dw, w)
        k_new = torch.stack([k.clone() for k, _ in rows]).contiguous()
        v_new = torch.stack([v.clone() for _, v in rows]).contiguous()
        dw.kv.k_new, dw.kv.v_new = k_new.data_ptr(), v_new.data_ptr()
    out = torch.empty_like(dw.q)
    ws = S.alloc_workspace(dw.shape, dw.kv, max(w.S, 1), KIND_CODE[kind])
    ws_dense = S.alloc_workspace(dw.shape, dw.kv, 1, S.SANTA_KIND_DENSE)
    plan = S.santa_plan_info(dw.shape, dw.kv, max(w.S, 1), KIND_CODE[kind])
    plan["path_name"] = {v: k for k, v in S.PATHS.items()}[plan["path"]]
    stream = torch.cuda.current_stream()
    mask = None
    if kind == "bernoulli":
        mask = torch.empty((w.B, w.Hkv, w.d), dtype=torch.uint8, device=dev)

    def step(idx_out=None):
        if kind == "systematic":
            S.santa_decode_systematic(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, idx_out, out, ws,
                                      stream)
        elif kind == "stratified":
            S.santa_decode_stratified(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, idx_out, out, ws,
                                      stream)
        elif kind == "bernoulli":
            S.santa_decode_bernoulli_qk(dw.q, dw.kt, dw.kv, dw.shape, w.scale, w.B_draws, w.mode,
                                        dw.u_q, w.S, dw.u, idx_out, mask, out, ws, stream)
        elif kind == "flash":
            S.santa_decode_flash(dw.q, dw.kv, dw.shape, w.scale, w.tile, w.S_tile, dw.u, idx_out,
                                 out, ws, stream)
        elif kind == "iid":
            S.santa_decode_iid(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, idx_out, out, ws, stream)
        else:
            S.santa_decode_dense(dw.q, dw.kv, dw.shape, w.scale, out, ws, stream)

    def dense_step():
        S.santa_decode_dense(dw.q, dw.kv, dw.shape, w.scale, out, ws_dense, stream)

    # ---- algorithmic bytes (untimed call with idx_out) ----
    qsz = 2 if w.dtype == "bf16" else 4            # q and out elements
    esz = 1 if w.kv_dtype == "fp8" else qsz        # cache elements
    L = w.ctx_len.astype(np.int64)
    k_bytes = int(L.sum()) * w.Hkv * w.d * esz
    uniq_rows = 0
    feat_frac = 1.0
    if kind != "dense":
        ns = w.S if kind != "flash" else ((w.n_max + w.tile - 1) // w.tile) * w.S_tile
        idx = torch.empty((w.B, w.Hq, ns), dtype=torch.int32, device=dev)
        step(idx)
        torch.cuda.synchronize()
        ix = idx.cpu().numpy().reshape(w.B, w.Hkv, w.G * ns)
        uniq_rows = int(sum(len(np.unique(ix[b, k][ix[b, k] >= 0]))
                            for b in range(w.B) for k in range(w.Hkv)))
        if kind == "bernoulli":
            m = mask.cpu().numpy()
            feat_frac = float(m.mean())
            k_bytes = int(sum(int(m[b].sum()) * int(L[b]) for b in range(w.B))) * esz
    v_bytes = (uniq_rows if kind != "dense" else int(L.sum()) * w.Hkv) * w.d * esz
    io_bytes = 2 * w.B * w.Hq * w.d * qsz + (w.u.nbytes if w.u is not None else 0)
    if w.kv_dtype == "fp8":
        io_bytes += w.k_scale.nbytes + w.v_scale.nbytes
    if kind == "bernoulli":
        io_bytes += w.u_q.nbytes
    alg_bytes = k_bytes + v_bytes + io_bytes
    dense_bytes = 2 * int(L.sum()) * w.Hkv * w.d * esz + 2 * w.B * w.Hq * w.d * qsz

    # ---- timing ----
    flush = torch.empty(int(args.flush_gib * (1 << 30)) // 4, dtype=torch.float32, device=dev)
    flush.zero_()
    flush_ro = torch.zeros(2 * flush.numel(), dtype=torch.float32, device=dev)

    def cold_cache():
        flush.add_(1.0)        # evicts L2 / Infinity Cache / TLB (paper's in-place update)
        flush_ro.sum()         # clean lines: the update's dirty lines are written back now

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def timed(fn, steps, warmup, cold=True):
        """Per-step times in µs as (call, kernel), from two passes of `steps`
        steps.  Pass 1: events recorded on the stream around the library call
        (includes launch latency; this is the step time).  Pass 2: events the
        library attaches to its own first dispatch and last completion
        (santa_time_next_call), i.e. the interval a kernel trace reports; the
        attachment itself adds latency to the call, hence the separate pass."""
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        call_evs = [(ev(), ev()) for _ in range(steps)]
        kern_evs = [(ev(), ev()) for _ in range(steps)]
        for a, b in kern_evs:  # creates the HIP events behind the attached pairs
            a.record(stream)
            b.record(stream)
        torch.cuda.synchronize()
        for a, b in call_evs:
            if cold:
                cold_cache()
            a.record(stream)
            fn()
            b.record(stream)
        for a, b in kern_evs:
            if cold:
                cold_cache()
            S.santa_time_next_call(a, b)
            fn()
        torch.cuda.synchronize()
        call = np.array([a.elapsed_time(b) * 1e3 for a, b in call_evs])
        kern = np.array([a.elapsed_time(b) * 1e3 for a, b in kern_evs])
        return call, kern

    torch.cuda.synchronize()
    wall0 = time.time()
    us, kus = timed(step, args.steps, args.warmup)
    wall = time.time() - wall0
    S.check_workspace(ws)  # every timed call's bounded waits completed
    print(f"[bench] {kind}: call mean {us.mean():.2f} us  median {np.median(us):.2f}  "
          f"min {us.min():.2f} | kernel mean {kus.mean():.2f} us", file=sys.stderr, flush=True)
    res = {}
    if not args.no_dense and kind != "dense":
        dus, dkus = timed(dense_step, args.steps, args.warmup)
        S.check_workspace(ws_dense)
        res["dense_us_per_step"] = round(float(dus.mean()), 3)
        res["dense_kernel_us"] = round(float(dkus.mean()), 3)
        res["dense_gbs"] = round(dense_bytes / (dus.mean() * 1e-6) / 1e9, 1)
        res["dense_kernel_gbs"] = round(dense_bytes / (dkus.mean() * 1e-6) / 1e9, 1)
        res["speedup_vs_dense"] = round(float(dus.mean() / us.mean()), 3)
        print(f"[bench] dense: call mean {dus.mean():.2f} us | kernel mean {dkus.mean():.2f} us",
              file=sys.stderr, flush=True)
    # attainable rate: the streaming-read calibration kernel on a buffer of the
    # step's algorithmic byte count, same cold-cache protocol and timing
    rd_bytes = (alg_bytes // 16) * 16
    rd_buf = torch.zeros(rd_bytes // 4, dtype=torch.float32, device=dev)
    rd_sink = torch.empty(S.STREAM_READ_GROUPS, dtype=torch.int32, device=dev)
    _, rdk = timed(lambda: S.santa_stream_read(rd_buf, rd_sink, stream), args.steps, args.warmup)
    del rd_buf
    rd_gbs = rd_bytes / (rdk.mean() * 1e-6) / 1e9
    print(f"[bench] streaming read of {rd_bytes} B: kernel mean {rdk.mean():.2f} us "
          f"({rd_gbs:.0f} GB/s)", file=sys.stderr, flush=True)
    if not args.profile:
        warm, wk = timed(step, args.steps, 2, cold=False)
        res["warm_us_per_step"] = round(float(warm.mean()), 3)
        res["warm_kernel_us"] = round(float(wk.mean()), 3)

    gbs = alg_bytes / (us.mean() * 1e-6) / 1e9
    if w.paged:
        cache_desc = (f"paged cache ({w.page_size}-token pages, shuffled table, "
                      f"ctx {int(w.ctx_len.min())}..{int(w.ctx_len.max())})")
    else:
        cache_desc = f"{args.layout} cache"
    if args.append:
        cache_desc += ", fused current-token append"
    if w.kv_dtype == "fp8":
        cache_desc += ", FP8 E4M3 K/V with per-(batch, KV head) scales"
    kgbs = alg_bytes / (kus.mean() * 1e-6) / 1e9
    line = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(float(us.mean()) / 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"cfg{args.cfg}: {w.kind} " +
                         (f"tile={w.tile} S_tile={w.S_tile}, " if kind == "flash" else f"S={w.S}, ") +
                         f"B={w.B}, Hq={w.Hq}, Hkv={w.Hkv}, d={w.d}, "
                         f"n_k={w.n_max}, {w.dtype}, {cache_desc}, cold cache "
                         f"({args.flush_gib:g} GiB update + {2 * args.flush_gib:g} GiB read per step)"),
            "path": plan["path_name"], "kernels": plan["kernels"],
            "batch": w.B, "n_k": w.n_max, "S": w.S, "kind": w.kind,
        },
        "us_per_step": round(float(us.mean()), 3),
        "us_median": round(float(np.median(us)), 3),
        "us_min": round(float(us.min()), 3),
        "kernel_us_per_step": round(float(kus.mean()), 3),
        "hbm_frac_of_peak": round(gbs / PEAK_HBM_GBS, 4),
        "bytes_touched": alg_bytes,
        "bytes_breakdown": {"k": k_bytes, "v_unique_rows": v_bytes, "q_out_u": io_bytes},
        "unique_v_rows": uniq_rows,
        "k_feature_fraction": round(feat_frac, 4),
        **res,
        "roofline": {
            "bound": "hbm",
            "kernel": plan["kernels"],
            "timing": ("HIP events the library attaches to its kernel dispatch "
                       "(santa_time_next_call), mean over the timed cold-cache steps"),
            "kernel_us": round(float(kus.mean()), 3),
            "achieved": round(kgbs, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(kgbs / PEAK_HBM_GBS, 4),
            "traffic": None,
        },
        "attainable_read": {
            "kernel": "k_stream_read (santa_stream_read)",
            "bytes": rd_bytes,
            "kernel_us": round(float(rdk.mean()), 3),
            "achieved": round(rd_gbs, 1),
            "unit": "GB/s",
            "frac_of_peak": round(rd_gbs / PEAK_HBM_GBS, 4),
            "step_frac": round(kgbs / rd_gbs, 4),
        },
        "timed_wall_s": round(wall, 3),
    }

    # counter-based traffic exists for each configuration's default workload
    if (args.cfg in TRAFFIC_FILES and args.B is None and args.S is None and args.kind is None
            and args.layout == "nhd" and args.path == "auto" and args.splits == 0
            and args.mode is None and args.B_draws is None and args.kv == "bf16"
            and not args.append):
        line["roofline"]["traffic"] = measured_traffic(line["roofline"]["kernel"],
                                                       TRAFFIC_FILES[args.cfg])
    if not args.no_cpu and not args.profile:
        line["cpu_baseline"] = cpu_baseline(w, kind, alg_bytes, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def flash_tile_budget(S_total: int, n_tiles: int) -> int:
    """Draws per tile for a total budget S spread over T tiles (S_tile ~ S/T,
    Sec. 3.3), rounded half up, at least one."""
    return max(1, (2 * int(S_total) + int(n_tiles)) // (2 * int(n_tiles)))


# Sources of each kernel family (the files its code is compiled from) for the
# hash recorded with the counter runs under profiles/: the shared headers, the
# launcher and the plan, plus the family's own header and instantiation units.
COMMON_SOURCES = ["include/santa.h", "csrc/santa_plan.h", "csrc/santa_device.h",
                  "csrc/santa_tiles.h", "csrc/santa_kernels.h", "csrc/santa_fused.h",
                  "csrc/santa_launch.hip", "csrc/santa_api.hip"]
FAMILY_SOURCES = {
    "k_fused_sampled": ["csrc/santa_sampled.h", "csrc/santa_sampled_*.hip"],
    "k_fused_dense": ["csrc/santa_dense.h", "csrc/santa_dense_*.hip"],
    "k_stream_cdf + k_value_heads": ["csrc/santa_stream.h", "csrc/santa_stream_*.hip"],
    "k_bern_stream + k_value_heads": ["csrc/santa_stream.h", "csrc/santa_stream_*.hip"],
    "k_row_sampled": ["csrc/santa_rows.h", "csrc/santa_rows_*.hip"],
    "k_row_flash": ["csrc/santa_rows.h", "csrc/santa_rows_*.hip"],
}
# counter runs per workload: (cfg, file under profiles/)
TRAFFIC_FILES = {2: "traffic_llama8b_32k_b1.json", 3: "traffic_llama8b_32k_b16.json",
                 4: "traffic_llama8b_paged_b64.json", 5: "traffic_llama8b_32k_b8_bernoulli.json"}


def kernel_source_hash(kernels: str) -> str:
    """Hash of the HIP sources of one kernel family (file names and contents),
    as recorded with the counter runs under profiles/."""
    import glob
    import hashlib
    h = hashlib.sha256()
    pkg = os.path.join(ROOT, "paper_2605_01910_amd")
    files = []
    for pat in COMMON_SOURCES + FAMILY_SOURCES[kernels]:
        base = ROOT if pat.startswith("include/") else pkg
        files += sorted(glob.glob(os.path.join(base, pat)))
    for f in files:
        h.update(os.path.relpath(f, ROOT).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernels: str, workload_file: str):
    """HBM bytes per call of the kernels `kernels` (one launch each) from the
    committed FETCH_SIZE / WRITE_SIZE runs, or None if there are none for this
    workload or the family's sources changed since they were taken."""
    path = os.path.join(ROOT, "profiles", workload_file)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    fam = rec.get("families", {}).get(kernels)
    if fam is None or fam.get("source_hash") != kernel_source_hash(kernels):
        return None
    return int(fam["bytes"])


def cpu_baseline(w, kind, alg_bytes, seconds):
    """The CPU oracle (float64 C, OpenMP over rows) timed on this host on full
    decode steps of the same workload, repeated for about `seconds`."""
    from oracle import oracle as O

    O.lib()
    reps, total, threads = 0, 0.0, 1
    t_end = time.time() + seconds
    while True:
        t0 = time.perf_counter()
        r = O.decode_workload(w, kind)
        total += time.perf_counter() - t0
        threads = r.threads
        reps += 1
        if time.time() >= t_end or reps >= 2000:
            break
    per = total / reps
    return {
        "value": round(alg_bytes / per / 1e9, 3),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"{reps} full decode step(s) of the same workload (all {w.B * w.Hq} rows), "
                   f"{per * 1e3:.1f} ms per step, float64, {threads} OpenMP threads, "
                   f"host nproc={os.cpu_count()}"),
        "ms_per_step": round(per * 1e3, 3),
    }


if __name__ == "__main__":
    main()
