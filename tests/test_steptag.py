"""Step-tag tracker of the controller (CPU only; host logic of the library).

* Scenarios written from the paper's rules (Section III-E): a failure in
  forward/backward resumes at step i, one in the optimizer step at i+1;
  stop only when every normal rank reported after the failure was detected;
  a data-parallel group with no live rank falls back to a checkpoint
  (Section III-G).
* A discrete-event simulation of training ranks with the barrier before the
  optimizer step and periodic heartbeats: whatever the failure time, the
  tracker never stops at a wrong step, never calls the state inconsistent,
  and stops at the step the failed rank's phase implies.
* The library equals the plain restatement in ``oracle/steptag.py`` on random
  event sequences, and donors are spread over the live ranks of each group.

The scenarios and the simulation run on both the library and the plain
restatement (through ``OracleTracker``), so they pin the restatement too;
tests/test_oracle_mutants.py plants mistakes in it that they must catch.
"""
import numpy as np
import pytest

from oracle.steptag import Cluster
from paper_2509_03047_amd import flashrestore as F


class OracleTracker:
    """The plain restatement behind the library's Tracker interface
    (decisions carry the action and the resume step only)."""

    cluster = Cluster

    def __init__(self, n_ranks, dp_group=None, timeout_s=10.0, now_s=0.0):
        groups = [0] * n_ranks if dp_group is None else [int(x) for x in dp_group]
        self.c = self.cluster(n_ranks, groups, timeout_s, now_s)

    def heartbeat(self, rank, tag, now):
        self.c.heartbeat(rank, tag, now)

    def report_failure(self, rank, now):
        self.c.report_failure(rank, now)

    def decide(self, now):
        action, step = self.c.decide(now)
        return {"action": action, "resume_step": step}

    def failed_ranks(self, now):
        return self.c.failed(now)

    def donors(self, now):
        return self.c.donors(now)


IMPLS = {"library": F.Tracker, "oracle": OracleTracker}


@pytest.fixture(params=sorted(IMPLS))
def make(request):
    return IMPLS[request.param]


def _same(d, expect: dict):
    """d agrees with every field of expect that it carries (the restatement
    reports no counts)."""
    return all(d[k] == v for k, v in expect.items() if k in d)


def test_no_failure_continues(make):
    t = make(4, None, 2.0, 0.0)
    for r in range(4):
        t.heartbeat(r, 3, 1.0)
    assert t.decide(1.5)["action"] == "continue"


def test_failure_in_forward_backward_resumes_at_i(make):
    t = make(4, [0, 0, 1, 1], 2.0, 0.0)
    for r in range(4):
        t.heartbeat(r, 5, 1.0)
    t.report_failure(2, 1.2)
    d = t.decide(1.3)
    assert _same(d, {"action": "wait", "n_waiting": 3})  # reports predate the failure
    for r in (0, 1, 3):
        t.heartbeat(r, 5, 1.5)  # blocked at the barrier before the optimizer step
    d = t.decide(1.6)
    assert _same(d, {"action": "stop_and_restore", "resume_step": 5, "n_failed": 1, "n_waiting": 0})
    assert t.donors(1.6) == [-1, -1, 3, -1]


def test_failure_in_optimizer_step_resumes_at_i_plus_1(make):
    t = make(3, None, 2.0, 0.0)
    for r in range(3):
        t.heartbeat(r, -1, 1.0)
    t.report_failure(0, 1.1)
    t.heartbeat(1, -1, 1.2)
    t.heartbeat(2, 6, 1.2)
    assert t.decide(1.3)["action"] == "wait"  # rank 1 still in its optimizer step
    t.heartbeat(1, 6, 1.4)
    d = t.decide(1.5)
    assert d["action"] == "stop_and_restore" and d["resume_step"] == 6


def test_stale_tag_from_before_the_failure_is_not_trusted(make):
    """A rank that reported i in forward and then entered its optimizer step
    must not be read as 'still at i'."""
    t = make(2, None, 5.0, 0.0)
    t.heartbeat(0, 9, 1.0)
    t.heartbeat(1, 9, 1.0)
    t.report_failure(1, 2.0)  # rank 1 died in its optimizer step of step 9
    assert t.decide(2.1)["action"] == "wait"
    t.heartbeat(0, 10, 2.3)
    assert t.decide(2.4)["resume_step"] == 10


def test_silent_rank_times_out(make):
    t = make(3, None, 1.0, 0.0)
    for r in range(3):
        t.heartbeat(r, 2, 0.5)
    t.heartbeat(0, 2, 1.2)
    t.heartbeat(1, 2, 1.2)
    assert t.decide(1.4)["action"] == "continue"
    assert t.failed_ranks(1.6) == [2]  # silent since 0.5, timeout 1.0
    assert t.decide(1.6)["action"] == "wait"  # detected at 1.5, reports at 1.2 are older
    t.heartbeat(0, 2, 1.7)
    t.heartbeat(1, 2, 1.7)
    assert t.decide(1.8)["action"] == "stop_and_restore"


def test_lost_group_falls_back_to_checkpoint(make):
    t = make(4, [0, 1, 0, 1], 5.0, 0.0)
    for r in range(4):
        t.heartbeat(r, 1, 0.1)
    t.report_failure(1, 0.2)
    t.report_failure(3, 0.2)
    assert t.decide(0.3)["action"] == "checkpoint_fallback"
    assert t.donors(0.3) == [-1, -1, -1, -1]


def test_disagreeing_fresh_tags_are_inconsistent(make):
    t = make(3, None, 5.0, 0.0)
    t.report_failure(2, 0.5)
    t.heartbeat(0, 4, 1.0)
    t.heartbeat(1, 7, 1.0)
    assert t.decide(1.1)["action"] == "inconsistent"


def test_donors_spread_over_live_ranks(make):
    g = [0] * 6 + [1] * 2
    t = make(8, g, 5.0, 0.0)
    for r in range(8):
        t.heartbeat(r, 0, 0.1)
    for r in (0, 1, 2, 7):
        t.report_failure(r, 0.2)
    d = t.donors(0.3)
    assert d[:3] == [3, 4, 5] and d[7] == 6
    assert all(d[r] == -1 for r in (3, 4, 5, 6))


def test_argument_errors():
    with pytest.raises(F.FlashRestoreError):
        F.Tracker(0)
    with pytest.raises(F.FlashRestoreError):
        F.Tracker(2, [0, 2], 1.0, 0.0)  # group id out of range
    with pytest.raises(F.FlashRestoreError):
        F.Tracker(2, None, 0.0, 0.0)
    t = F.Tracker(2, None, 1.0, 0.0)
    with pytest.raises(F.FlashRestoreError):
        t.heartbeat(2, 0, 0.1)
    with pytest.raises(F.FlashRestoreError):
        t.heartbeat(0, -2, 0.1)


# ------------------------------------------------------------ simulation


def simulate(rng, n_ranks, groups, failures, steps=12, hb=0.25):
    """Rank timelines under the paper's protocol.  failures: {rank: time}.
    Returns per-rank lists of (time, tag) changes and the step each failure
    implies (the paper's rule from the failed rank's phase)."""
    fwd = rng.uniform(1.0, 2.0, size=(steps, n_ranks))
    opt = rng.uniform(0.2, 0.5, size=(steps, n_ranks))
    start = np.zeros(n_ranks)
    changes = {r: [(0.0, 0)] for r in range(n_ranks)}
    implied = {}
    for i in range(steps):
        end_fwd = start + fwd[i]
        release = end_fwd.max()
        # the barrier completes only if every rank is alive when it releases
        if any(tf <= release for tf in failures.values()):
            for f, tf in failures.items():
                if f not in implied:
                    implied[f] = i if tf < release else i + 1
            break
        for r in range(n_ranks):
            changes[r].append((release, -1))
            changes[r].append((release + opt[i, r], i + 1))
        for f, tf in failures.items():
            if f not in implied and tf < release + opt[i, f]:
                implied[f] = i + 1  # died inside its optimizer step of step i
        if len(implied) == len(failures) and failures:
            break
        start = release + opt[i]
    return changes, implied


def tag_at(changes, t):
    tag = changes[0][1]
    for when, v in changes:
        if when <= t:
            tag = v
    return tag


def check_simulation(seed, make):
    """One simulated failure (seed) against a tracker made by `make`: the
    tracker never calls the state inconsistent, stops only at the step the
    failed rank's phase implies, and stops at all when a replica is left.
    Returns False when the failure falls past the simulated horizon."""
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(2, 9))
    n_groups = int(rng.integers(1, n + 1))
    groups = [r % n_groups for r in range(n)]
    f = int(rng.integers(0, n))
    tf = float(rng.uniform(0.5, 15.0))
    changes, implied = simulate(rng, n, groups, {f: tf})
    if f not in implied:
        return False
    expect = implied[f]
    has_replica = sum(1 for r in range(n) if groups[r] == groups[f]) > 1
    hb = 0.25
    timeout = 1.0
    report = bool(rng.integers(0, 2))
    t = make(n, groups, timeout, 0.0)
    phase = rng.uniform(0, hb, size=n)
    events = []
    for r in range(n):
        k = phase[r]
        while k < tf + 8.0:
            if not (r == f and k >= tf):
                events.append((k, "hb", r))
            k += hb
    if report:
        events.append((tf + float(rng.uniform(0.0, 0.8)), "fail", f))
    polls = np.arange(0.0, tf + 8.0, 0.05)
    events += [(float(p), "poll", -1) for p in polls]
    events.sort()
    stops = []
    for when, kind, r in events:
        if kind == "hb":
            t.heartbeat(r, tag_at(changes[r], when), when)
        elif kind == "fail":
            t.report_failure(r, when)
        else:
            d = t.decide(when)
            if not has_replica:  # the failed rank is alone in its group
                assert d["action"] in ("continue", "checkpoint_fallback")
                continue
            assert d["action"] != "inconsistent", when
            if d["action"] == "stop_and_restore":
                assert d["resume_step"] == expect, (when, tf, expect)
                stops.append(when)
    if has_replica:
        assert stops, "no stop decision"
    return True


@pytest.mark.parametrize("seed", range(40))
def test_simulated_failures_resume_at_the_papers_step(seed, make):
    if not check_simulation(seed, make):
        pytest.skip("failure after the simulated horizon")


def test_library_equals_plain_rules_on_random_events():
    rng = np.random.default_rng(7)
    for _ in range(300):
        n = int(rng.integers(1, 7))
        groups = [int(x) for x in rng.integers(0, n, size=n)]
        timeout = float(rng.uniform(0.5, 2.0))
        t = F.Tracker(n, groups, timeout, 0.0)
        oc = Cluster(n, groups, timeout, 0.0)
        now = 0.0
        for _ in range(40):
            now += float(rng.exponential(0.3))
            u = rng.random()
            r = int(rng.integers(0, n))
            if u < 0.6:
                tag = int(rng.choice([-1, 3, 4, 5]))
                t.heartbeat(r, tag, now)
                oc.heartbeat(r, tag, now)
            elif u < 0.7:
                t.report_failure(r, now)
                oc.report_failure(r, now)
            d = t.decide(now)
            assert (d["action"], d["resume_step"]) == oc.decide(now)
            assert t.failed_ranks(now) == oc.failed(now)
            assert t.donors(now) == oc.donors(now)


def test_donors_into_equals_donors():
    t = F.Tracker(6, [0, 0, 0, 1, 1, 1], 5.0, 0.0)
    for r in range(6):
        t.heartbeat(r, 2, 0.1)
    t.report_failure(1, 0.2)
    t.report_failure(4, 0.2)
    out = np.full(6, 99, np.int32)
    assert t.donors_into(0.3, out).tolist() == t.donors(0.3)


def test_binding_checks_host_arrays():
    """The binding refuses host arrays of the wrong length or type before
    the library reads them."""
    with pytest.raises(ValueError):
        F.Tracker(4, [0, 1], 1.0, 0.0)  # group array shorter than the ranks
    t = F.Tracker(3, None, 1.0, 0.0)
    with pytest.raises(ValueError):
        t.donors_into(0.0, np.zeros(2, np.int32))
    with pytest.raises(ValueError):
        t.donors_into(0.0, np.zeros(3, np.int64))
    L = F.Layout3D(2, 1, 2, 1, 0)
    with pytest.raises(ValueError):
        L.donors_into(np.zeros(4, np.uint8), np.zeros(3, np.int32))
    with pytest.raises(ValueError):
        L.donors_into(np.zeros(4, np.int32), np.zeros(4, np.int32))
