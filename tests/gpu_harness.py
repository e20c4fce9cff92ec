"""Run a group decode on the GPU through the C ABI and compare with the oracle.

Inputs are staged on the device in windows of steps, so workloads whose
per-step inputs exceed device memory still run in the launch configuration the
benchmark uses.  Outputs of selected steps are copied back for comparison.
"""

import sys
import time

import numpy as np

from oracle import attend_slot, simulate_group
from paper_2506_22950_amd.group import context_for, decode_group, plan_steps, probe_group, schedulers_for
from workload import Workload
from workload.staging import DeviceInputs


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_gpu_group(cfg, policy, capture=lambda step: True, split=0, window=1024, wl=None, stop_after=None, reuse=0,
                  probe=None, inspect=None, kv_fp8=False, exchange=None, entry="decode_step", scale=0.0,
                  step_split=None, probe_entry="probe_step"):
    """Group decode through the C ABI.  reuse = k runs the probe phase of prefix
    reuse first; if `probe` is a dict it receives 'log' (probe step log) and
    'captured' (the O buffer [L, batch, Hq, d] after every probe step).
    inspect(ctx, step, log) is called after every decode step; kv_fp8 stores the
    KV cache as E4M3; exchange sets the partial exchange mode (default: the
    library's); entry names the C call that decodes each layer; scale is the
    context's softmax scale (0: 1/sqrt(head_dim)); step_split sets the work
    split of step launches (default: the library's); probe_entry is the C call
    of the probe phase (infs_probe_step per layer, or infs_probe_step_layers)."""
    import torch

    assert torch.cuda.is_available(), "GPU test needs a GPU"
    wl = wl or Workload(cfg)
    plog = []
    log = plan_steps(cfg, wl.L, policy, wl.L_hat, stop_after=stop_after, reuse=reuse, probe_log=plog)
    dev = DeviceInputs(wl)
    stream = torch.cuda.current_stream()
    ctx = context_for(cfg, stream=stream, split_tokens=split, probe_tokens=reuse, kv_fp8=kv_fp8, scale=scale)
    if exchange is not None:
        ctx.set_exchange(exchange)
    if step_split is not None:
        ctx.set_step_split(step_split)
    keep = []
    for p in range(cfg.num_prompts):
        for layer in range(cfg.layers):
            k, v = dev.prefix(layer, p)
            keep.append((k, v))
            ctx.prefill_shared(p, layer, cfg.prompt_lens[p], k, v)
    L, S, Hq, Hkv, d = cfg.layers, cfg.num_slots, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    es = cfg.elem_bytes
    o = torch.empty((L, S, Hq, d), dtype=torch.float32, device="cuda")
    o_ptr = o.data_ptr()
    n = len(log)
    win = {"w0": 0, "w1": 0, "bufs": None}

    def provide(k, layer):
        if not (win["w0"] <= k < win["w1"]):
            win["bufs"] = None
            w1 = min(n, k + window)
            win["bufs"] = dev.stage(log, k, w1)
            win["w0"], win["w1"] = k, w1
            win["ptrs"] = [t.data_ptr() for t in win["bufs"]]
        j = (k - win["w0"]) * L + layer
        qp, kp, vp = win["ptrs"]
        return (qp + j * S * Hq * d * es, kp + j * S * Hkv * d * es, vp + j * S * Hkv * d * es,
                o_ptr + layer * S * Hq * d * 4)

    captured = {}

    def after(step):
        if capture(step):
            captured[step] = o.cpu().numpy()
        if inspect is not None:
            inspect(ctx, step, log)

    t0 = time.time()
    if reuse:
        pq, pk, pv = dev.stage(plog, 0, len(plog))
        W = pq.shape[2]
        po = torch.zeros((L, W, Hq, d), dtype=torch.float32, device="cuda")
        pcap = {}

        def pprovide(j, p, first, n, layer):
            return (pq[j, layer].data_ptr(), pk[j, layer].data_ptr(), pv[j, layer].data_ptr(), po[layer].data_ptr())

        def pafter(j):
            pcap[j] = po.cpu().numpy()

        nprobe = probe_group(ctx, wl.L, reuse, L, pprovide, after_step=pafter, entry=probe_entry)
        assert nprobe == len(plog)
        if probe is not None:
            probe["log"], probe["captured"] = plog, pcap
    steps = decode_group(ctx, schedulers_for(cfg, policy, wl.L_hat), wl.L, L, provide, after_step=after,
                         stop_after=stop_after, reuse=reuse, entry=entry)
    torch.cuda.synchronize()
    tokens = np.stack([ctx.sample_tokens(p) for p in range(cfg.num_prompts)])
    stats = ctx.get_stats()
    ctx.destroy()
    say(f"  [{cfg.name} {policy}] {steps} steps, {n * L} launches in {time.time() - t0:.1f}s")
    return wl, log, steps, captured, tokens, stats


class _PrefixCache:
    """The workload with its prefix rows memoised (they are the same for every step)."""

    def __init__(self, wl):
        self._wl, self.cfg, self._cache = wl, wl.cfg, {}

    def prefix_kv(self, layer, p):
        if (layer, p) not in self._cache:
            self._cache[(layer, p)] = self._wl.prefix_kv(layer, p)
        return self._cache[(layer, p)]

    def suffix_kv(self, layer, p, i, t):
        return self._wl.suffix_kv(layer, p, i, t)

    def query(self, layer, p, i, t):
        return self._wl.query(layer, p, i, t)


def check_against_oracle(cfg, wl, log, captured, layers=None, tol=None, kv_fp8=False, scale=None):
    """Max abs error over every captured live (step, slot, layer) output; idle rows must be 0.
    kv_fp8: the oracle rounds keys and values to E4M3 as the FP8 cache stores them; scale: the
    softmax scale (None: 1/sqrt(head_dim))."""
    tol = tol if tol is not None else (1e-2 if cfg.dtype == "bf16" else 1e-5)
    layers = range(cfg.layers) if layers is None else layers
    wl = _PrefixCache(wl)
    worst = 0.0
    checked = 0
    for k, o in captured.items():
        for s, e in enumerate(log[k]):
            if e is None:
                assert not o[:, s].any(), f"idle slot {s} at step {k} has nonzero output"
                continue
            p, i, t = e
            for layer in layers:
                ref = attend_slot(wl, layer, p, i, t, scale=scale, kv_fp8=kv_fp8)
                err = float(np.abs(o[layer, s].astype(np.float64) - ref).max())
                assert np.isfinite(o[layer, s]).all()
                if err > worst:
                    worst = err
                assert err <= tol, f"step {k} slot {s} sample {i} t {t} layer {layer}: max abs err {err:.3g} > {tol}"
                checked += 1
    return worst, checked


def oracle_dynamic_log(cfg, wl, target):
    """Step log of dynamic-slot sampling from the oracle simulator (per prompt)."""
    from oracle import simulate_dynamic
    res = [simulate_dynamic(wl.L[p], cfg.slots_per_prompt, target) for p in range(cfg.num_prompts)]
    out = []
    for k in range(max(r.steps for r in res)):
        row = []
        for p, r in enumerate(res):
            for ls in range(cfg.slots_per_prompt):
                e = r.log[k][ls] if k < r.steps else None
                row.append(None if e is None else (p, e[0], e[1]))
        out.append(tuple(row))
    return out


def oracle_log(cfg, wl, policy, reuse=0):
    total, res = simulate_group(wl.L, cfg.slots_per_prompt, policy, wl.L_hat, reuse=reuse)
    m = cfg.slots_per_prompt
    out = []
    for k in range(total):
        row = []
        for p, r in enumerate(res):
            for ls in range(m):
                e = r.log[k][ls] if k < r.steps else None
                row.append(None if e is None else (p, e[0], e[1]))
        out.append(tuple(row))
    return out


def sample_steps(log, every=13, edge=4, refills=None):
    """Steps to check: every `every`-th, the first and last `edge`, and the steps
    where some slot decodes its first token (just refilled) -- all of them, or
    `refills` of them spread evenly."""
    n = len(log)
    keep = set(range(0, n, every)) | set(range(min(edge, n))) | set(range(max(0, n - edge), n))
    fills = [k for k, row in enumerate(log) if any(e is not None and e[2] == 1 for e in row)]
    if refills is not None and len(fills) > refills:
        fills = [fills[int(i)] for i in np.linspace(0, len(fills) - 1, refills)]
    keep.update(fills)
    return keep
