"""Plain restatement of the restore planner's layout rules for the tests.
TEST INFRASTRUCTURE ONLY.  Rank order t fastest, then data index d, then
pipeline index p; d = s + shard * q; ranks with equal (t, p, s) are replicas.
"""


def coords(tp, pp, dp, shard, rank):
    t = rank % tp
    d = (rank // tp) % dp
    p = rank // (tp * dp)
    return t, p, d, d % shard, d // shard


def replicas(tp, pp, dp, shard, rank):
    t, p, d, s, q = coords(tp, pp, dp, shard, rank)
    return [t + tp * (s + shard * qq + dp * p) for qq in range(dp // shard)]


def donors(tp, pp, dp, shard, failed):
    world = tp * pp * dp
    out = [-1] * world
    served = {}
    for r in range(world):
        if r not in failed:
            continue
        live = [x for x in sorted(replicas(tp, pp, dp, shard, r)) if x not in failed]
        key = tuple(sorted(replicas(tp, pp, dp, shard, r)))
        if live:
            k = served.get(key, 0)
            out[r] = live[k % len(live)]
            served[key] = k + 1
    return out


def shard_range(numel, shard, s):
    """Element range [lo, hi) of shard s and the padded total."""
    n = sum(numel)
    unit = 8 * shard
    npad = -(-n // unit) * unit
    e = npad // shard
    return s * e, (s + 1) * e, npad
