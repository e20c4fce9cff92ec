"""Benchmark: shared-prefix continuous-sampling group decode on one MI355X.

One benchmark step is one whole group decode of the throughput workload
(28 layers, 16 query / 8 KV heads, head_dim 128, a 2048-token shared prompt,
G=64 samples on m=16 slots, lognormal lengths, SJF refill on noisy predicted
lengths, bf16 K/V): prefill of the shared prompt KV for every layer, then every
running step (refill, one decode_step per layer, end_step, retire) until all 64
samples are done.  All inputs are synthetic and staged in HBM before timing.

Prints one JSON line with tokens/s (value), the roofline of the decode kernel
(algorithmic bytes per launch over its average duration, timed with HIP events
on the library's stream in a separate pass), and the CPU oracle timed on a
bounded sample of the same workload.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
COPY_CAL_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "{kernel}_traffic_{workload}.txt")
MFMA_FILE = os.path.join(ROOT, "profiles", "{kernel}_mfma_{workload}.txt")
CALIB_LIB = os.path.join(ROOT, "paper_2506_22950_amd", "libinfs_calib.so")
PEAK_MFMA_BF16_TFLOPS = 2500.0
SIMDS = 1024  # 256 compute units x 4 SIMDs
XCDS = 8
MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", "GRBM_GUI_ACTIVE")
KERNEL_SOURCES = tuple("paper_2506_22950_amd/csrc/" + f for f in (
    "decode.h", "layers.h", "step_plan.h", "kernels.h", "plan.h", "kernels.hip", "inst_wave_f32_d64.hip",
    "inst_wave_f32_d128.hip",
    "inst_wave_bf16_d64.hip", "inst_wave_bf16_d128.hip", "inst_mfma_d64.hip", "inst_mfma_d128a.hip",
    "inst_mfma_d128b.hip", "inst_kv8a.hip", "inst_kv8b.hip"))
METRIC = "generated tokens/sec per group decode + achieved HBM TB/s vs peak, 1 MI355X"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _code_only(text):
    """Source text without comments and with whitespace runs collapsed, so that a
    comment-only edit keeps the hash (and the counter summaries tied to it)."""
    import re

    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash():
    """SHA-256 over the code (comments stripped) of the decode kernel sources."""
    import hashlib

    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()


def _read_summary(path):
    """key = value lines of a committed counter summary, or None when there is
    none or the kernel source has changed since it was taken."""
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as fh:
        for ln in fh:
            if "=" in ln and not ln.startswith("#"):
                k, v = ln.split("=", 1)
                kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return kv


KERNELS = {"decode_step_layers": "layers_kernel", "decode_step": "decode_kernel"}


def entry_launches(cfg, steplog, entry):
    """Kernel launches of one group decode: one per running step for the step
    launch through every layer, one per layer and step otherwise."""
    return len(steplog) * (1 if entry == "decode_step_layers" else cfg.layers)


def read_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary of this
    workload, or None when there is none or the kernel source has changed since."""
    kv = _read_summary(TRAFFIC_FILE.format(kernel=kernel, workload=workload))
    return None if kv is None else float(kv["traffic_bytes_per_launch"])


def read_mfma(workload, kernel):
    """MFMA counter summary of this workload's launches of `kernel` (or None)."""
    return _read_summary(MFMA_FILE.format(kernel=kernel, workload=workload))


def mfma_flops(cfg, steplog, split=256, nj=None):
    """MFMA flops issued by all launches of a group decode (2 flops per
    multiply-add of every 16x16x32 tile issued), every KV head, every layer:
    (prefix) per prompt with a live slot, S^T = K Q^T and O^T = V^T P^T over
    the padded row tile (m * hpk rows padded to 16/32/64/128) and 32-token
    blocks; (responses, bf16 and E4M3 pages) per live slot, per wavefront of
    each split-K item, per 32-token page pair of its stored tokens (the newest
    token is folded in apart): two S^T tiles of head_dim / 32 steps, then
    head_dim / 16 O^T tiles and one row-sum tile, each 16 columns wide with hpk
    of them carrying query rows.  The items are the per-layer launch's chunks
    of `split` tokens, or, with nj (work-groups per KV head of a step launch),
    the items the library's step-launch plan gives each step
    (infs_step_split_plan).  fp32 contexts issue no MFMA."""
    if cfg.dtype != "bf16":
        return 0.0
    rows = cfg.slots_per_prompt * cfg.hpk
    pad = 16 if rows <= 16 else 32 if rows <= 32 else 64 if rows <= 64 else 128
    d = cfg.head_dim
    per_prompt = [4 * pad * (-(-plen // 32) * 32) * d * cfg.num_kv_heads for plen in cfg.prompt_lens]
    tile = 2 * 16 * 16 * 32
    per_pair = (2 * (d // 32) + d // 16 + 1) * tile
    sub = split // 4
    pairs_memo = {}

    def pairs(length):  # page pairs the wavefronts of one slot multiply
        if length not in pairs_memo:
            n, last = 0, length - 1
            for t0 in range(0, length, split):
                t1 = min(t0 + split, length)
                for w in range(4):
                    w0 = min(t0 + w * sub, t1)
                    w1 = min(w0 + sub, t1)
                    te = last if w0 <= last < w1 else w1
                    n += -(-(te - w0) // 32) if te > w0 else 0
            pairs_memo[length] = n
        return pairs_memo[length]

    def wave_pairs(length, ranges):  # ranges: each wavefront's [w0, w1) token range
        last = length - 1
        n = 0
        for w0, w1 in ranges:
            te = last if w0 <= last < w1 else w1
            n += -(-(te - w0) // 32) if te > w0 else 0
        return n

    def piece_pairs(length, n):  # near-equal page ranges, as the step launch cuts them
        pages = -(-length // 16)
        ranges = []
        for c in range(n):
            pg0, pg1 = c * pages // n, (c + 1) * pages // n
            ppw = -(-(pg1 - pg0) // 4)
            t1 = min(pg1 * 16, length)
            for w in range(4):
                w0 = min((pg0 + w * ppw) * 16, t1)
                ranges.append((w0, min(w0 + ppw * 16, t1)))
        return wave_pairs(length, ranges)

    plan = None
    if nj is not None:
        from paper_2506_22950_amd import infs

        scmax = -(-cfg.max_suffix_len // split)

        def plan(row):
            # the library's rule: the per-layer launch's 128-token prefix chunks unless they would
            # give some producer two items, then 256-token chunks (MFMA tiles, bf16 or E4M3 cache)
            lens = [e[2] if e is not None else 0 for e in row]
            live = {e[0] for e in row if e is not None}
            npi = sum(-(-cfg.prompt_lens[p] // 128) for p in live)
            r0, _ = infs.step_split_plan(nj, lens, npi, 128, split, scmax, mode=0)
            psplit = 256 if (r0["items"] > r0["n_suf"] or r0["n_pre"] < npi) else 128
            npi = sum(-(-cfg.prompt_lens[p] // psplit) for p in live)
            roles, pieces = infs.step_split_plan(nj, lens, npi, psplit, split, scmax)
            return roles["cut"], pieces

    total = 0
    for row in steplog:
        total += sum(per_prompt[p] for p in {e[0] for e in row if e is not None})
        cut, pieces = plan(row) if plan is not None else (0, None)
        if cut:
            n = sum(piece_pairs(e[2], int(pieces[s])) for s, e in enumerate(row) if e is not None)
        else:
            n = sum(pairs(e[2]) for e in row if e is not None)
        total += n * per_pair * cfg.num_kv_heads
    return total * cfg.layers


def read_ceiling(torch, stream, nbytes, launches=200, pool_bytes=2 << 30, read_budget=40 << 30):
    """The one-launch read-bandwidth reference: a plain streaming-read kernel
    (libinfs_calib.so) over `nbytes` (rounded down to a multiple of 16 KiB),
    launched back to back over distinct buffers of a pool of at least 2 GiB and
    two launches (so no launch finds its bytes in the 256 MB last-level cache),
    timed like the decode
    launches: HIP events on `stream` around all launches, divided by their
    number.  Best of 256, 512 and 1024 work-groups.
    Returns (bytes, us per launch, work-groups)."""
    import ctypes

    if not os.path.exists(CALIB_LIB):
        raise RuntimeError(f"{CALIB_LIB} is missing: build it with `python -m paper_2506_22950_amd.build`")
    fn = ctypes.CDLL(CALIB_LIB).infs_calib_stream_read
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    nb = nbytes // (16 << 10) * (16 << 10)
    nbuf = max(2, pool_bytes // nb)  # a step launch through every layer can read more than the pool
    launches = max(5, min(launches, read_budget // nb))  # at most ~40 GiB read per grid size
    pool = torch.empty(nbuf * nb, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1024, dtype=torch.int32, device="cuda")
    with torch.cuda.stream(stream):
        pool.fill_(1)
    best = None
    for blocks in (256, 512, 1024):
        def launch(i):
            rc = fn(pool.data_ptr() + (i % nbuf) * nb, nb, blocks, stream.cuda_stream, sink.data_ptr())
            if rc != 0:
                raise RuntimeError(f"infs_calib_stream_read failed: hipError {rc}")

        for i in range(5):
            launch(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(launches):
            launch(i)
        e1.record(stream)
        e1.synchronize()
        us = e0.elapsed_time(e1) * 1000.0 / launches
        if best is None or us < best[1]:
            best = (nb, us, blocks)
    del pool
    return best


def copy_calibration(torch):
    """Three device-to-device copies of COPY_CAL_BYTES: the plain copy kernel whose
    FETCH_SIZE / WRITE_SIZE readings scale the decode kernel's."""
    src = torch.empty(COPY_CAL_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def _pmc_rows(path, counter):
    import csv
    import glob

    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {path}")
    rows = []
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    rows.append(r)
    return rows


def summarize_pmc(workload, fetch_dir, write_dir, entry="decode_step_layers"):
    """Text summary of two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) of
    `bench.py --steps 1 --warmup 0 --no-kernel-timing --no-cpu-baseline --copy-calibration`:
    per-launch HBM traffic of the entry's kernel, each counter scaled by its
    reading for the calibration copy of known size."""
    from paper_2506_22950_amd.group import plan_steps
    from workload import Workload, get_config

    kernel = KERNELS[entry]
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _pmc_rows(d, counter)
        dec = [float(r["Counter_Value"]) for r in rows if kernel in r["Kernel_Name"]]
        cps = [r for r in rows if "copyBuffer" in r["Kernel_Name"]]
        gmax = max(int(r["Grid_Size"]) for r in cps)
        cal = [float(r["Counter_Value"]) for r in cps if int(r["Grid_Size"]) == gmax]
        if len(cal) < 3 or not dec:
            raise SystemExit(f"{counter}: {len(cal)} calibration copies, {len(dec)} decode launches")
        cal_kib = sorted(cal)[len(cal) // 2]
        scale = COPY_CAL_BYTES / (cal_kib * 1024.0)
        out[counter] = (len(dec), sum(dec) / len(dec), cal_kib, scale)
    cfg = get_config(workload)
    wl = Workload(cfg)
    steplog = plan_steps(cfg, wl.L, cfg.policy, wl.L_hat)
    launches = entry_launches(cfg, steplog, entry)
    alg = algorithmic_bytes(cfg, steplog) / launches
    nf, fk, cf, sf = out["FETCH_SIZE"]
    nw, wk, cw, sw = out["WRITE_SIZE"]
    if nf != launches or nw != launches:
        raise SystemExit(f"expected {launches} {kernel} launches, got {nf} / {nw}")
    fetch_b, write_b = fk * 1024.0 * sf, wk * 1024.0 * sw
    lines = [
        f"kernel_source_sha256 = {kernel_source_hash()}",
        f"workload = {workload}",
        f"kernel = {kernel}",
        f"launches = {launches}",
        f"copy_bytes = {COPY_CAL_BYTES}",
        f"copy_fetch_kib = {cf:.1f}",
        f"copy_write_kib = {cw:.1f}",
        f"fetch_scale = {sf:.4f}",
        f"write_scale = {sw:.4f}",
        f"fetch_kib_per_launch = {fk:.1f}",
        f"write_kib_per_launch = {wk:.1f}",
        f"fetch_bytes_per_launch = {fetch_b:.0f}",
        f"write_bytes_per_launch = {write_b:.0f}",
        f"traffic_bytes_per_launch = {fetch_b + write_b:.0f}",
        f"alg_bytes_per_launch = {alg:.0f}",
        f"traffic_over_alg = {(fetch_b + write_b) / alg:.3f}",
    ]
    return "\n".join(lines)


def summarize_mfma(workload, pmc_dir, entry="decode_step_layers"):
    """Text summary of one rocprofv3 --pmc run of MFMA_COUNTERS over
    `bench.py --steps 1 --warmup 1 --no-kernel-timing --no-cpu-baseline`:
    MFMA work and MFMA busy cycles of the entry's kernel per launch.  Counter
    values are summed over their hardware instances (shader engines, XCDs)."""
    from paper_2506_22950_amd.group import plan_steps
    from workload import Workload, get_config

    kernel = KERNELS[entry]
    per = {}
    for counter in MFMA_COUNTERS:
        vals = [float(r["Counter_Value"]) for r in _pmc_rows(pmc_dir, counter) if kernel in r["Kernel_Name"]]
        if not vals:
            raise SystemExit(f"{counter}: no {kernel} rows under {pmc_dir}")
        per[counter] = (len(vals), sum(vals) / len(vals))
    cfg = get_config(workload)
    wl = Workload(cfg)
    steplog = plan_steps(cfg, wl.L, cfg.policy, wl.L_hat)
    launches = entry_launches(cfg, steplog, entry)
    counts = {n for n, _ in per.values()}
    if len(counts) != 1 or next(iter(counts)) % launches:
        raise SystemExit(f"expected whole group decodes of {launches} launches per counter, got {sorted(counts)}")
    decodes = next(iter(counts)) // launches
    mops = per["SQ_INSTS_VALU_MFMA_MOPS_BF16"][1]
    busy = per["SQ_VALU_MFMA_BUSY_CYCLES"][1]
    cu_busy_quads = per["SQ_BUSY_CU_CYCLES"][1]
    gui = per["GRBM_GUI_ACTIVE"][1] / XCDS
    nj = None
    if entry == "decode_step_layers":  # the step launch's plan depends on the device's work-group count
        from paper_2506_22950_amd.group import context_for

        ctx = context_for(cfg)
        nj = ctx.step_launch_workgroups // cfg.num_kv_heads
        ctx.destroy()
    expect = mfma_flops(cfg, steplog, nj=nj) / launches
    lines = [
        f"kernel_source_sha256 = {kernel_source_hash()}",
        f"workload = {workload}",
        f"kernel = {kernel}",
        f"launches = {launches} per group decode, {decodes} group decodes profiled",
        f"mfma_mops_bf16_per_launch = {mops:.1f}",
        f"mfma_flops_per_launch = {mops * 512:.0f}",
        f"expected_mfma_flops_per_launch = {expect:.0f}",
        f"mfma_busy_cycles_per_launch = {busy:.1f}",
        f"cu_busy_cycles_per_launch = {cu_busy_quads * 4:.1f}",
        f"gpu_active_cycles_per_launch = {gui:.1f}",
        f"mfma_busy_over_active_simd_cycles = {busy / (gui * SIMDS):.5f}",
        f"mfma_busy_over_busy_cu_simd_cycles = {busy / (cu_busy_quads * 4 * 4):.5f}",
    ]
    return "\n".join(lines)


def summarize_counter(counter, pmc_dir, entry="decode_step_layers"):
    """Mean of one --pmc counter per launch of the entry's kernel (summed over
    its hardware instances), with the number of launches it covers."""
    kernel = KERNELS[entry]
    vals = [float(r["Counter_Value"]) for r in _pmc_rows(pmc_dir, counter) if kernel in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"{counter}: no {kernel} rows under {pmc_dir}")
    return f"{kernel} {counter}: {sum(vals) / len(vals):.1f} per launch over {len(vals)} launches"


def summarize_stats(workload, stats_dir, bench_out, entry="decode_step_layers", command=""):
    """Kernel statistics table of a `rocprofv3 --kernel-trace --stats` run of
    `bench.py --steps K --warmup W` (without --no-kernel-timing): the run decodes
    the group W + K + 2 times (warmup, timed, then the HIP-event and the
    device-clock timing passes); the header says so and quotes the command and
    the JSON line that run printed."""
    import csv
    import glob

    files = glob.glob(os.path.join(stats_dir, "**", "*kernel_stats.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one kernel_stats.csv under {stats_dir}, found {len(files)}")
    with open(files[0]) as fh:
        rows = list(csv.DictReader(fh))
    with open(bench_out) as fh:
        line = [ln.strip() for ln in fh if ln.strip().startswith("{")][-1]
    b = json.loads(line)
    passes = b["warmup"] + b["steps"] + 2
    kernel = KERNELS[entry]
    main = [r for r in rows if kernel in r["Name"]]
    if not main:
        raise SystemExit(f"no {kernel} row in {files[0]}")
    out = [f"# rocprofv3 kernel statistics, workload {workload}: {passes} whole group decodes",
           f"# ({b['warmup']} warmup, {b['steps']} timed, then the HIP-event and the device-clock timing passes)",
           "# of the command below, run on one MI355X from the repository root after: cd /tmp && export TMPDIR=/tmp",
           f"#   {command}" if command else "#   (command not given)",
           f"#   python3 bench.py --workload {workload} --entry {'step' if entry == 'decode_step_layers' else 'layer'}"
           f" --summarize-stats <stats dir> <bench output>",
           "# bench.py line printed by that same run (its launch times include the profiler's per-dispatch overhead):",
           "#   " + line, "",
           f"{'kernel':<62}{'calls':>8}{'avg_us':>10}{'min_us':>10}{'max_us':>10}{'total_ms':>11}{'pct':>7}"]
    for r in rows:
        n = r["Name"]
        short = n if len(n) <= 60 else n[:57] + "..."
        out.append(f"{short:<62}{int(r['Calls']):>8}{float(r['AverageNs']) / 1e3:>10.3f}{float(r['MinNs']) / 1e3:>10.3f}"
                   f"{float(r['MaxNs']) / 1e3:>10.3f}{float(r['TotalDurationNs']) / 1e6:>11.2f}{float(r['Percentage']):>7.2f}")
    out += ["", f"{kernel} full name: " + main[0]["Name"],
            f"{kernel} launches per group decode: {b['roofline']['launches'] if b.get('roofline') else 'n/a'}; "
            f"average by the profiler {float(main[0]['AverageNs']) / 1e3:.3f} us, by HIP events in that run "
            f"{b['roofline']['avg_launch_us'] if b.get('roofline') else 'n/a'} us"]
    return "\n".join(out)


def schedule_table(n_groups=64, G=32, m=4, cap=1024):
    """Running steps of the refill policies (Table 2 style) and the length bias
    of dynamic-slot sampling (Table 1 style), from the library's host scheduler
    in dry-run mode (no GPU): n_groups groups of G samples on m slots per
    length setting; steps summed over the groups.  The post-hoc optimum
    (Infinite*) comes from the library's exact branch and bound
    (infs_sched_optimum); longest-first list scheduling on the true lengths is
    only an upper bound on it."""
    import math

    from paper_2506_22950_amd.group import plan_steps
    from workload import SCHEDULER_STUDY, get_config, scheduler_study_lengths, scheduler_study_stream

    cfg = get_config("tiny_f32").with_(layers=1, samples_per_prompt=G, slots_per_prompt=m, max_suffix_len=cap)
    from paper_2506_22950_amd import infs

    rows = [("naive micro groups", "naive", "pred"), ("fixed-slot", "fixed_row", "pred"),
            ("FPTAS only", "fptas", "pred"), ("SJF only", "sjf", "pred"), ("FPTAS + SJF", "fptas_sjf", "pred"),
            ("post-hoc LPT (true lengths)", "lpt", "true")]
    out = [f"{n_groups} groups of G={G} on m={m} slots, lengths capped at {cap}, "
           f"predictions L*exp(N(0, 0.2^2)); running steps summed over the groups (ratio to fixed-slot); "
           f"mean length of the G samples kept per group"]
    for k, (label, mu, sigma) in enumerate(SCHEDULER_STUDY):
        L, pred = scheduler_study_lengths(mu, sigma, n_groups, G, cap=cap, seed=k)
        tot = {}
        for _, policy, key in rows:
            tot[policy] = sum(len(plan_steps(cfg, L[n:n + 1], policy, (L if key == "true" else pred)[n:n + 1]))
                              for n in range(n_groups))
        stream = scheduler_study_stream(mu, sigma, L, 8 * G, cap=cap, seed=k)
        dcfg = cfg.with_(samples_per_prompt=stream.shape[1])
        dyn_steps, dyn_len = 0, []
        for n in range(n_groups):
            acc = []
            dyn_steps += len(plan_steps(dcfg, stream[n:n + 1], "fifo", None, stop_after=G, accepted=acc))
            dyn_len.extend(int(stream[n, i]) for i in acc[0])
        lb = sum(max(math.ceil(int(L[n].sum()) / m), int(L[n].max())) for n in range(n_groups))
        opt = [infs.sched_optimum(L[n], m) for n in range(n_groups)]
        opt_best, opt_low = sum(o[0] for o in opt), sum(o[1] for o in opt)
        unsolved = sum(o[0] != o[1] for o in opt)
        out.append(f"\n{label}: mean length {L.mean():.0f}")
        base = tot["fixed_row"]
        for name, policy, _ in rows:
            out.append(f"  {name:30s} {tot[policy]:8d}  (x{tot[policy] / base:.2f})  mean length {L.mean():6.1f}")
        out.append(f"  {'dynamic-slot (stream, first G)':30s} {dyn_steps:8d}  (x{dyn_steps / base:.2f})  "
                   f"mean length {sum(dyn_len) / len(dyn_len):6.1f}")
        if unsolved == 0:
            out.append(f"  {'post-hoc optimum (Infinite*)':30s} {opt_best:8d}  (x{opt_best / base:.2f})  "
                       f"mean length {L.mean():6.1f}  (proven for all {n_groups} groups)")
        else:
            out.append(f"  {'post-hoc optimum (Infinite*)':30s} {opt_low:8d}..{opt_best}  "
                       f"({n_groups - unsolved} of {n_groups} groups proven; the rest bounded)")
        out.append(f"  {'lower bound max(sum/m, max)':30s} {lb:8d}  (x{lb / base:.2f})")
    return "\n".join(out)


def algorithmic_bytes(cfg, steplog, kv_bytes=None):
    """Algorithmic HBM bytes of all decode launches, from the step log alone:
    prefix K/V once per prompt with a live slot, each live slot's stored
    response K/V, the new token's K/V read and append write, Q read and fp32 O
    write.  kv_bytes: stored bytes per K/V element (default: the input size)."""
    kvb = cfg.elem_bytes if kv_bytes is None else kv_bytes
    kvrow = cfg.num_kv_heads * cfg.head_dim * kvb
    kvrow_in = cfg.num_kv_heads * cfg.head_dim * cfg.elem_bytes
    total = 0.0
    for row in steplog:
        live_prompts = {e[0] for e in row if e is not None}
        b = sum(2.0 * cfg.prompt_lens[p] * kvrow for p in live_prompts)
        for e in row:
            if e is not None:
                b += (2.0 * (e[2] - 1) * kvrow + 2.0 * kvrow_in + 2.0 * kvrow
                      + cfg.num_q_heads * cfg.head_dim * (cfg.elem_bytes + 4))
        total += b
    return total * cfg.layers


STAGE_BUDGET_BYTES = 160 << 30  # staged per-step inputs beyond this are cycled through a window


ENTRIES = {"step": "decode_step_layers", "layer": "decode_step"}
PROBE_ENTRIES = {"step": "probe_step_layers", "layer": "probe_step"}


class Bench:
    def __init__(self, cfg_name, split=0, reuse=0, kv_fp8=False, entry="step", overrides=None, probe_entry="layer"):
        import numpy as np
        import torch

        from paper_2506_22950_amd import infs
        from paper_2506_22950_amd.group import context_for, plan_steps
        from workload import Workload, get_config
        from workload.staging import DeviceInputs

        self.np, self.torch = np, torch
        self.entry = ENTRIES[entry]
        self.probe_entry = PROBE_ENTRIES[probe_entry]
        infs.load()
        cfg = get_config(cfg_name, **(overrides or {}))
        self.cfg = cfg
        t0 = time.time()
        self.wl = wl = Workload(cfg)
        self.reuse = reuse
        self.plog = []
        self.log = plan_steps(cfg, wl.L, cfg.policy, wl.L_hat, reuse=reuse, probe_log=self.plog)
        self.naive_steps = len(plan_steps(cfg, wl.L, "naive", wl.L_hat, reuse=reuse))
        # Infinite*: the post-hoc optimum of the true lengths; prompts run side by side on their own slots
        opt = [infs.sched_optimum(wl.L[p], cfg.slots_per_prompt) for p in range(cfg.num_prompts)]
        self.optimum_steps = max(o[0] for o in opt) if all(o[0] == o[1] for o in opt) else None
        dev = DeviceInputs(wl)
        self.prefix = [[dev.prefix(l, p) for l in range(cfg.layers)] for p in range(cfg.num_prompts)]
        per_step = cfg.layers * cfg.num_slots * (cfg.num_q_heads + 2 * cfg.num_kv_heads) * cfg.head_dim * cfg.elem_bytes
        # Every step's Q / new K / new V rows are staged in HBM before timing.  A
        # workload whose rows exceed the budget stages a window of steps and step k
        # reads window row k mod W: the same launches and bytes, other input values
        # (bench outputs are not compared; the parity tests use the true rows).
        self.window = min(len(self.log), max(1, STAGE_BUDGET_BYTES // per_step))
        self.q, self.k, self.v = dev.stage(self.log, 0, self.window)
        if reuse:
            self.pq, self.pk, self.pv = dev.stage(self.plog, 0, len(self.plog))
            self.po = torch.empty((cfg.layers,) + tuple(self.pq.shape[2:4]) + (cfg.head_dim,), dtype=torch.float32,
                                  device="cuda")
        del dev
        torch.cuda.synchronize()
        self.stream = torch.cuda.current_stream()
        self.ctx = context_for(cfg, stream=self.stream, split_tokens=split, probe_tokens=reuse, kv_fp8=kv_fp8)
        self.kv_bytes = 1 if kv_fp8 else cfg.elem_bytes
        L, S, Hq, Hkv, d, es = cfg.layers, cfg.num_slots, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, cfg.elem_bytes
        self.o = torch.empty((L, S, Hq, d), dtype=torch.float32, device="cuda")
        self.qp, self.kp, self.vp, self.op = (self.q.data_ptr(), self.k.data_ptr(), self.v.data_ptr(),
                                              self.o.data_ptr())
        self.sq, self.skv, self.so = S * Hq * d * es, S * Hkv * d * es, S * Hq * d * 4
        self.L = L
        self.tokens = wl.total_tokens
        self.alg_bytes = algorithmic_bytes(cfg, self.log, self.kv_bytes)
        self.probe_alg_bytes = algorithmic_bytes(cfg, self.plog, self.kv_bytes) if reuse else 0.0
        log(f"setup {time.time() - t0:.1f}s: {len(self.log)} steps ({cfg.policy}) vs {self.naive_steps} naive, "
            f"{self.tokens} tokens, staged {(self.q.numel() + self.k.numel() + self.v.numel()) * es / 2**30:.1f} GiB"
            + ("" if self.window == len(self.log) else f" ({self.window} of {len(self.log)} steps, cycled)"))

    def provide(self, k, layer):
        j = (k % self.window) * self.L + layer
        return (self.qp + j * self.sq, self.kp + j * self.skv, self.vp + j * self.skv, self.op + layer * self.so)

    def provide_probe(self, j, p, first, n, layer):
        return (self.pq[j, layer].data_ptr(), self.pk[j, layer].data_ptr(), self.pv[j, layer].data_ptr(),
                self.po[layer].data_ptr())

    def prefill(self):
        cfg, ctx = self.cfg, self.ctx
        ctx.reset()
        for p in range(cfg.num_prompts):
            for layer in range(cfg.layers):
                k, v = self.prefix[p][layer]
                ctx.prefill_shared(p, layer, cfg.prompt_lens[p], k, v)

    def probe(self):
        """The probe phase of prefix reuse (nothing without it)."""
        from paper_2506_22950_amd.group import probe_group

        if self.reuse:
            probe_group(self.ctx, self.wl.L, self.reuse, self.cfg.layers, self.provide_probe, entry=self.probe_entry)

    def decode(self):
        from paper_2506_22950_amd.group import decode_group, schedulers_for

        cfg = self.cfg
        return decode_group(self.ctx, schedulers_for(cfg, cfg.policy, self.wl.L_hat), self.wl.L, cfg.layers,
                            self.provide, reuse=self.reuse, entry=self.entry)

    def group_decode(self):
        """One benchmark step: prefill every layer, the probe phase (with prefix
        reuse), then decode the whole group."""
        self.prefill()
        self.probe()
        return self.decode()

    def check_bookkeeping(self, steps):
        np = self.np
        assert steps == len(self.log), (steps, len(self.log))
        for p in range(self.cfg.num_prompts):
            assert np.array_equal(self.ctx.sample_tokens(p), self.wl.L[p]), "token counters"

    def host_cost(self):
        """Host time per decode call of the entry: the whole group replayed on a
        dry-run context (the Python step loop, ctypes and the library's host
        planning and bookkeeping; no device work, no launch).  Returns
        (us per call, calls per group decode)."""
        from paper_2506_22950_amd.group import context_for, decode_group, schedulers_for

        cfg = self.cfg
        ctx = context_for(cfg, dry_run=True, probe_tokens=self.reuse)
        for p in range(cfg.num_prompts):
            for layer in range(cfg.layers):
                ctx.prefill_shared(p, layer, cfg.prompt_lens[p], None, None)
        nothing = (None, None, None, None)
        t0 = time.perf_counter()
        steps = decode_group(ctx, schedulers_for(cfg, cfg.policy, self.wl.L_hat), self.wl.L, cfg.layers,
                             lambda k, layer: nothing, reuse=self.reuse, entry=self.entry)
        dt = time.perf_counter() - t0
        ctx.destroy()
        calls = steps * (1 if self.entry == "decode_step_layers" else cfg.layers)
        return dt * 1e6 / calls, calls

    def event_timing(self):
        """One more whole group decode: HIP events on the library's stream (the
        torch stream the context was created on) around the decode launches
        only (prefill and probe phase outside).  Returns (ms, launches)."""
        torch = self.torch
        self.prefill()
        self.probe()
        before = self.ctx.get_stats().launches
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        self.decode()
        e1.record(self.stream)
        e1.synchronize()
        return e0.elapsed_time(e1), self.ctx.get_stats().launches - before

    def kernel_timing(self):
        """One more whole group decode with the library's device-clock timing on:
        the summed kernel body time of the decode launches (first block start to
        last block end of each).  With prefix reuse the probe launches are timed
        in a pass of their own: returns (decode timing, probe timing or None),
        each (ms, region_ms, launches, library alg bytes, library launches)."""
        self.prefill()
        probe = None
        if self.reuse:
            self.ctx.timing_begin()
            self.probe()
            ms, region_ms, n = self.ctx.timing_end()
            st = self.ctx.get_stats()
            probe = (ms, region_ms, n, st.alg_bytes, st.launches)
        before = self.ctx.get_stats()
        self.ctx.timing_begin()
        self.decode()
        ms, region_ms, n = self.ctx.timing_end()
        st = self.ctx.get_stats()
        return (ms, region_ms, n, st.alg_bytes - before.alg_bytes, st.launches - before.launches), probe


CPU_POOL_MAX = 16  # worker processes at most (a host's CPU share per GPU)


def _oracle_worker_init(cfg_name, overrides):
    global _ORACLE_WL
    from threadpoolctl import threadpool_limits

    from workload import Workload, get_config

    threadpool_limits(limits=1)
    _ORACLE_WL = Workload(get_config(cfg_name, **overrides))


def _oracle_worker(unit):
    """One (step, layer) unit of the CPU baseline: the float64 oracle for every
    live slot of that step at that layer.  Returns its wall seconds."""
    from oracle import attend_slot

    layer, entries = unit
    t0 = time.perf_counter()
    for p, i, t in entries:
        attend_slot(_ORACLE_WL, layer, p, i, t)
    return time.perf_counter() - t0


def cpu_sample_steps(steplog):
    """Steps of the CPU baseline's sample: every step = 0 mod 97, the first and
    last 8, and every step in which some slot decodes its first token (a refill)."""
    n = len(steplog)
    keep = {k for k in range(n) if k % 97 == 0} | set(range(min(8, n))) | set(range(max(0, n - 8), n))
    keep |= {k for k, row in enumerate(steplog) if any(e is not None and e[2] == 1 for e in row)}
    return sorted(keep)


def step_flops(cfg, row):
    """Attention flops of one step at one layer: 4 * Hq * d * (P + t) per live slot."""
    return sum(4.0 * cfg.num_q_heads * cfg.head_dim * (cfg.prompt_lens[e[0]] + e[2]) for e in row if e is not None)


def cpu_baseline(bench):
    """The float64 oracle on the host's cores (a pool of spawned worker processes,
    one BLAS thread each) over a sample of the workload -- steps = 0 mod 97,
    the first and last 8, every refill step, on layers 0, L/2 and L-1 -- with the
    full run's time extrapolated by the ratio of attention flops."""
    import multiprocessing as mp
    from dataclasses import asdict

    from threadpoolctl import threadpool_info

    cfg, steplog = bench.cfg, bench.log
    steps = cpu_sample_steps(steplog)
    layers = sorted({0, cfg.layers // 2, cfg.layers - 1})
    units = [(layer, [e for e in steplog[k] if e is not None]) for k in steps for layer in layers]
    sample_flops = sum(step_flops(cfg, steplog[k]) for k in steps) * len(layers)
    total_flops = sum(step_flops(cfg, row) for row in steplog) * cfg.layers
    cores = len(os.sched_getaffinity(0))
    workers = max(1, min(cores, CPU_POOL_MAX))
    base = asdict(get_config_default(cfg.name))
    overrides = {k: v for k, v in asdict(cfg).items() if base.get(k) != v}
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers, initializer=_oracle_worker_init, initargs=(cfg.name, overrides)) as pool:
        pool.map(_oracle_worker, units[:workers])  # warm the workers up (pools drawn, imports done)
        t0 = time.perf_counter()
        busy = sum(pool.map(_oracle_worker, units, chunksize=1))
        wall = time.perf_counter() - t0
    blas = sorted({str(i.get("internal_api")) for i in threadpool_info()})
    est = wall * total_flops / sample_flops
    return {
        "value": round(bench.tokens / est, 4),
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": (f"{len(steps)} of {len(steplog)} steps (= 0 mod 97, first and last 8, every refill step) x layers "
                   f"{layers}: {len(units)} (step, layer) units, {sample_flops / 1e12:.3f} of {total_flops / 1e12:.2f} "
                   f"TFLOP; {wall:.1f} s wall on {workers} worker processes ({busy:.1f} s busy), extrapolated to the "
                   f"whole group by the flop ratio; float64 numpy, 1 BLAS thread per worker"),
        "host_cpus": cores,
        "blas": blas,
        "blas_threads_per_worker": 1,
    }


def get_config_default(name):
    from workload import get_config

    return get_config(name)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="qwen3_1p7b_g64")
    ap.add_argument("--split", type=int, default=0)
    ap.add_argument("--G", type=int, help="samples per prompt (overrides the workload's)")
    ap.add_argument("--m", type=int, help="slots per prompt")
    ap.add_argument("--prompt-len", help="prompt lengths, comma separated (one per prompt)")
    ap.add_argument("--policy", choices=("naive", "fixed_row", "fifo", "sjf", "fptas", "fptas_sjf", "lpt"),
                    help="refill policy")
    ap.add_argument("--seed", type=int, help="seed of the length, prediction and Q/K/V draws")
    ap.add_argument("--dtype", choices=("bf16", "f32"), help="storage type of Q, K, V")
    ap.add_argument("--layers", type=int, help="number of layers")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--reuse", type=int, default=0, metavar="K",
                    help="prefix reuse: every sample decodes K probe tokens first (Section 4); default 0")
    ap.add_argument("--kv-fp8", action="store_true",
                    help="store the KV cache as E4M3 (halves the K/V bytes; not the headline configuration)")
    ap.add_argument("--exchange", type=int, choices=(0, 1), default=None,
                    help="partial exchange: 0 through the coherence point, 1 through the XCD's L2 "
                         "(default: the library's choice)")
    ap.add_argument("--probe-entry", choices=tuple(PROBE_ENTRIES), default="layer",
                    help="probe phase of --reuse: layer = one launch per layer (infs_probe_step, the default: "
                         "faster for a 64-sample batch), step = one launch per probe step (infs_probe_step_layers)")
    ap.add_argument("--step-split", type=int, choices=(0, 1), default=None,
                    help="work split of step launches: 1 near-equal response pieces (the library's default), "
                         "0 the per-layer launch's chunks")
    ap.add_argument("--entry", choices=tuple(ENTRIES), default="step",
                    help="step: one launch per running step through every layer (infs_decode_step_layers); "
                         "layer: one launch per layer (infs_decode_step)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run three 1 GiB device copies first (counter calibration for --summarize-pmc)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the traffic summary of two rocprofv3 --pmc output folders and exit")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("STATS_DIR", "BENCH_OUT"),
                    help="print the kernel statistics of a rocprofv3 --kernel-trace --stats run of bench.py "
                         "(BENCH_OUT: the JSON line that run printed)")
    ap.add_argument("--summarize-counter", nargs=2, metavar=("COUNTER", "PMC_DIR"),
                    help="print the mean per launch of one counter of a rocprofv3 --pmc run")
    ap.add_argument("--profile-command", default="",
                    help="the profiled command line, quoted in the --summarize-stats header")
    ap.add_argument("--summarize-mfma", metavar="PMC_DIR",
                    help="print the MFMA summary of a rocprofv3 --pmc output folder and exit")
    ap.add_argument("--schedules", action="store_true",
                    help="print the running steps of the refill policies (host only, no GPU) and exit")
    args = ap.parse_args()
    if args.summarize_counter:
        print(summarize_counter(args.summarize_counter[0], args.summarize_counter[1], entry=ENTRIES[args.entry]))
        return
    if args.summarize_stats:
        print(summarize_stats(args.workload, *args.summarize_stats, entry=ENTRIES[args.entry],
                              command=args.profile_command))
        return
    if args.summarize_pmc:
        print(summarize_pmc(args.workload, *args.summarize_pmc, entry=ENTRIES[args.entry]))
        return
    if args.summarize_mfma:
        print(summarize_mfma(args.workload, args.summarize_mfma, entry=ENTRIES[args.entry]))
        return
    if args.schedules:
        print(schedule_table())
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library decodes a group on one GPU and has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        copy_calibration(torch)
    overrides = {k: v for k, v in (("samples_per_prompt", args.G), ("slots_per_prompt", args.m),
                                    ("policy", args.policy), ("seed", args.seed), ("dtype", args.dtype),
                                    ("layers", args.layers)) if v is not None}
    if args.prompt_len:
        overrides["prompt_lens"] = tuple(int(x) for x in args.prompt_len.split(","))
    b = Bench(args.workload, split=args.split, reuse=args.reuse, kv_fp8=args.kv_fp8, entry=args.entry,
              overrides=overrides, probe_entry=args.probe_entry)
    if args.exchange is not None:
        b.ctx.set_exchange(args.exchange)
    if args.step_split is not None:
        b.ctx.set_step_split(args.step_split)

    for w in range(args.warmup):
        t0 = time.time()
        steps = b.group_decode()
        torch.cuda.synchronize()
        b.check_bookkeeping(steps)
        log(f"warmup {w}: {time.time() - t0:.2f}s")

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        steps = b.group_decode()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    b.check_bookkeeping(steps)
    ms_per_step = elapsed * 1000.0 / args.steps
    value = b.tokens * args.steps / elapsed
    log(f"timed {args.steps} group decodes: {ms_per_step:.1f} ms each, {value:.0f} tokens/s, "
        f"end-to-end {(b.alg_bytes + b.probe_alg_bytes) / (ms_per_step / 1e3) / 1e9:.0f} GB/s algorithmic")

    roof, probe = None, None
    if not args.no_kernel_timing:
        ev_ms, ev_n = b.event_timing()
        (ms, region_ms, n, alg, launches), ptiming = b.kernel_timing()
        assert n == launches == ev_n, (n, launches, ev_n)
        rel = abs(alg - b.alg_bytes) / b.alg_bytes
        assert rel < 1e-9, f"library and step-log byte counts differ: {alg} vs {b.alg_bytes}"
        avg_us = ev_ms * 1000.0 / n
        body_us = ms * 1000.0 / n
        per_launch = alg / n
        achieved = per_launch / (avg_us * 1e-6) / 1e9
        kernel = KERNELS[b.entry]
        traffic = (read_traffic(args.workload, kernel) if not (args.reuse or args.kv_fp8 or args.exchange is not None
                                                               or args.step_split is not None or args.split
                                                               or overrides) else None)
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                "kernel": kernel,
                "launches": n, "avg_launch_us": round(avg_us, 3),
                "alg_bytes_per_launch": round(per_launch),
                "timing": "HIP events on the kernels' stream around all decode launches of one group decode, "
                          "divided by their number",
                "launch_covers": ("every layer of one running step" if b.entry == "decode_step_layers"
                                  else "one layer of one running step"),
                "kernel_body_us": round(body_us, 3),
                "kernel_body_timing": "device wall clock, first block start to last block end, averaged per launch",
                "body_achieved": round(per_launch / (body_us * 1e-6) / 1e9, 1)}
        mf = (read_mfma(args.workload, kernel) if not (args.reuse or args.kv_fp8 or args.split or overrides
                                                       or args.step_split is not None) else None)
        if mf is not None:
            fl = float(mf["mfma_flops_per_launch"])
            roof["mfma"] = {"kernel": f"{kernel} (prefix and response contractions)", "flops_per_launch": round(fl),
                            "tflops": round(fl / (avg_us * 1e-6) / 1e12, 2), "peak_tflops": PEAK_MFMA_BF16_TFLOPS,
                            "frac": round(fl / (avg_us * 1e-6) / 1e12 / PEAK_MFMA_BF16_TFLOPS, 5),
                            "busy_over_active": float(mf["mfma_busy_over_active_simd_cycles"]),
                            "source": os.path.relpath(MFMA_FILE.format(kernel=kernel, workload=args.workload), ROOT)}
        cb, cus, cblocks = read_ceiling(torch, b.stream, int(per_launch))
        cgbs = cb / (cus * 1e-6) / 1e9
        roof["read_ceiling"] = {"kernel": "plain streaming read, one launch (libinfs_calib.so)", "bytes": cb,
                                "work_groups": cblocks, "avg_launch_us": round(cus, 3), "achieved": round(cgbs, 1),
                                "frac": round(cgbs / PEAK_HBM_GBS, 4)}
        roof["frac_of_read_ceiling"] = round(achieved / cgbs, 4)
        log(f"read ceiling: {cb / 1e6:.2f} MB in {cus:.2f} us per launch ({cblocks} work-groups) -> {cgbs:.0f} GB/s")
        log(f"kernel: {n} launches, {avg_us:.2f} us per launch by HIP events, {per_launch / 1e6:.2f} MB/launch -> "
            f"{achieved:.0f} GB/s; kernel body {body_us:.2f} us (device clock)")
        if ptiming is not None:
            pms, pregion, pn, palg, plaunch = ptiming
            assert pn == plaunch, (pn, plaunch)
            assert abs(palg - b.probe_alg_bytes) <= 1e-9 * b.probe_alg_bytes, (palg, b.probe_alg_bytes)
            pavg = pms * 1000.0 / pn
            pper = palg / pn
            pach = pper / (pavg * 1e-6) / 1e9
            rows = b.ctx.probe_batch * b.cfg.hpk
            probe = {"kernel": ("layers_kernel (probe step launches through every layer, %d rows per KV head)" % rows
                                if b.probe_entry == "probe_step_layers" else
                                "decode_kernel (probe launches, one per layer, %d rows per KV head)" % rows),
                     "probe_tokens": args.reuse, "launches": pn, "avg_launch_us": round(pavg, 3),
                     "alg_bytes_per_launch": round(pper), "achieved": round(pach, 1), "unit": "GB/s",
                     "frac": round(pach / PEAK_HBM_GBS, 4), "phase_ms": round(pregion, 2)}
            log(f"probe: {pn} launches, avg {pavg:.2f} us, {pper / 1e6:.2f} MB/launch -> {pach:.0f} GB/s")

    host_us, host_calls = b.host_cost()
    log(f"host: {host_us:.1f} us per {b.entry} call (dry-run replay), {host_calls} calls per group decode")
    cpu = None if args.no_cpu_baseline else cpu_baseline(b)
    cfg = b.cfg
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": cfg.name,
            "layers": cfg.layers, "q_heads": cfg.num_q_heads, "kv_heads": cfg.num_kv_heads,
            "head_dim": cfg.head_dim, "prompt_len": list(cfg.prompt_lens), "G": cfg.samples_per_prompt,
            "m": cfg.slots_per_prompt, "policy": cfg.policy, "decode_steps": len(b.log),
            "naive_decode_steps": b.naive_steps, "optimum_decode_steps": b.optimum_steps,
            "generated_tokens": b.tokens,
            "alg_bytes_per_group": round(b.alg_bytes),
            "end_to_end_alg_GBps": round((b.alg_bytes + b.probe_alg_bytes) / (ms_per_step / 1e3) / 1e9, 1),
            "probe_tokens": args.reuse, "probe_steps": len(b.plog),
            "kv_cache": "e4m3" if args.kv_fp8 else cfg.dtype,
            "staged_steps": b.window,
            "exchange": {0: "coherence point", 1: "xcd l2"}[b.ctx.exchange_mode()],
            "entry": b.entry,
            "step_split": {0: "per-layer chunks", 1: "response pieces"}[1 if args.step_split is None
                                                                          else args.step_split],
            "overrides": {k: (list(v) if isinstance(v, tuple) else v) for k, v in overrides.items()},
        },
        "roofline": roof,
        "probe": probe,
        "host": {"us_per_call": round(host_us, 2), "calls_per_group_decode": host_calls,
                 "timing": "the group replayed on a dry-run context: Python step loop, ctypes and the library's "
                           "host planning, no device work"},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
