"""Pure-Python brute force used to pin the oracle on tiny shapes.

It gathers every key, value and query row one at a time straight from the
input generator's row addresses and sums with math.fsum, sharing nothing with
the oracle beyond the generator itself.
"""

import math


def brute_attend_slot(wl, l, p, i, t, h):
    c = wl.cfg
    hpk = c.num_q_heads // c.num_kv_heads
    g = h // hpk
    scale = 1.0 / math.sqrt(c.head_dim)
    q = [float(x) for x in wl.values("q", wl.query_index(l, p, i, [t - 1]))[0, h]]
    rows = list(wl.prefix_index(l, p)) + [int(wl.suffix_index(l, p, i, [j])[0]) for j in range(t)]
    scores, vals = [], []
    for r in rows:
        k = [float(x) for x in wl.values("k", [r])[0, g]]
        vals.append([float(x) for x in wl.values("v", [r])[0, g]])
        scores.append(math.fsum(a * b for a, b in zip(q, k)) * scale)
    mx = max(scores)
    e = [math.exp(s - mx) for s in scores]
    z = math.fsum(e)
    return [math.fsum(e[j] * vals[j][c_] for j in range(len(rows))) / z for c_ in range(c.head_dim)]
