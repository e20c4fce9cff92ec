"""Put a workload's inputs in device memory (torch is used for memory only).

The pools of Q/K/V rows are uploaded once; the per-step inputs of a group
decode are then gathered on the device into contiguous [steps, layers, S, H, d]
buffers, following a step log (which sample and position each slot decodes at
each step).  bf16 rows are kept as raw 16-bit patterns (torch.int16), fp32 rows
as float32.
"""

import numpy as np


class DeviceInputs:
    def __init__(self, wl, device="cuda"):
        import torch

        self.torch = torch
        self.wl = wl
        self.cfg = wl.cfg
        self.device = device
        conv = (lambda a: torch.from_numpy(a.view(np.int16))) if self.cfg.dtype == "bf16" else torch.from_numpy
        self.pool = {k: conv(np.ascontiguousarray(wl.pool(k))).to(device) for k in ("q", "k", "v")}

    def prefix(self, layer, prompt):
        """Prompt K and V of one layer, [P, Hkv, d] contiguous on the device."""
        idx = self.torch.from_numpy(self.wl.prefix_index(layer, prompt)).to(self.device)
        return self.pool["k"][idx].contiguous(), self.pool["v"][idx].contiguous()

    def indices(self, log, step0, step1):
        """Pool row indices [n, L, S] of Q and of the new K/V rows for steps [step0, step1);
        each log row lists, per slot (or probe batch position), (prompt, sample, t) or None."""
        c, wl = self.cfg, self.wl
        # rows are as wide as the widest step of the window (slots, or a probe batch)
        n, S = step1 - step0, max([c.num_slots] + [len(log[k]) for k in range(step0, step1)])
        qi = np.zeros((n, c.layers, S), dtype=np.int64)
        ki = np.zeros((n, c.layers, S), dtype=np.int64)
        # Group the (slot, step) entries by sample so each sample's rows come from one call.
        per_sample = {}
        for k in range(step0, step1):
            for s, e in enumerate(log[k]):
                if e is not None:
                    p, i, t = e
                    per_sample.setdefault((p, i), []).append((k - step0, s, t - 1))
        for (p, i), ents in per_sample.items():
            ks = np.array([e[0] for e in ents])
            ss = np.array([e[1] for e in ents])
            ts = np.array([e[2] for e in ents])
            for layer in range(c.layers):
                qi[ks, layer, ss] = wl.query_index(layer, p, i, ts)
                ki[ks, layer, ss] = wl.suffix_index(layer, p, i, ts)
        return qi, ki

    def stage(self, log, step0, step1):
        """(q, k_new, v_new) device tensors [n, L, S, H, d] for steps [step0, step1)."""
        torch = self.torch
        qi, ki = self.indices(log, step0, step1)
        qi = torch.from_numpy(qi).to(self.device)
        ki = torch.from_numpy(ki).to(self.device)
        return self.pool["q"][qi], self.pool["k"][ki], self.pool["v"][ki]
