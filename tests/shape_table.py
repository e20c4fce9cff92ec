"""Every decode kernel instantiation the library builds, each with a small
workload that selects it.

Selection (infs_create): the prefix runs on MFMA tiles iff the type is bf16 and
a prompt has at least 16 query rows per KV head (m * hpk); the row tile is the
smallest of 8/16 (wavefront path) or 16/32/64/128 (MFMA) that holds them.  The
probe launches of prefix reuse use the decode kernel's path with
probe_batch * hpk rows.  A bf16 wavefront tile of 16 rows with 8 query heads
per KV head is reached only that way (m = 1 decodes 8 rows, a probe batch of 2
samples 16)."""

from workload import get_config

HPKS = (1, 2, 4, 8)


def _entries():
    out = []
    for bf16 in (False, True):
        for d in (64, 128):
            for hpk in HPKS:
                for pr in (8, 16):
                    out.append((bf16, d, hpk, False, pr, False))
    for d in (64, 128):
        for hpk in HPKS:
            for pr in (16, 32, 64, 128):
                if not (pr == 128 and hpk == 1):
                    out.append((True, d, hpk, True, pr, False))
    for hpk in HPKS:
        for pr in (16, 32, 64, 128):
            if not (pr == 128 and hpk == 1):
                out.append((True, 128, hpk, True, pr, True))
    return out


ENTRIES = _entries()


def case_for(entry):
    """(config, probe_tokens, expected kernel info) for one instantiation: one
    layer, 2 KV heads, a 70-token prompt (ragged 32-token block), m slots and
    m + 5 samples of 1..30 tokens."""
    bf16, d, hpk, mfma, pr, kv8 = entry
    probe = 0
    if mfma:
        m = pr // hpk
    elif pr == 8:
        m = 8 // hpk
    elif not bf16:
        m = 16 // hpk
    elif hpk < 8:
        m = 15 // hpk
    else:
        m, probe = 1, 3  # reached by the probe kernel only
    cfg = get_config("tiny_f32").with_(
        name=f"shape_{'bf16' if bf16 else 'f32'}_d{d}_hpk{hpk}_{'mfma' if mfma else 'wave'}{pr}{'_kv8' if kv8 else ''}",
        layers=1, num_q_heads=2 * hpk, num_kv_heads=2, head_dim=d, prompt_lens=(70,), samples_per_prompt=m + 5,
        slots_per_prompt=m, length_dist=("uniform", 1, 30), max_suffix_len=30, dtype="bf16" if bf16 else "f32",
        seed=11 + hpk)
    want = {"bf16": int(bf16), "head_dim": d, "hpk": hpk, "kv_fp8": int(kv8)}
    if probe:
        want.update(mfma=0, prefix_rows=8, probe_mfma=0, probe_prefix_rows=pr)
    else:
        want.update(mfma=int(mfma), prefix_rows=pr)
    return cfg, probe, want


def case_id(entry):
    return case_for(entry)[0].name
