"""Plain restatement of the controller's step-tag rules (Section III-E) for
the tests.  TEST INFRASTRUCTURE ONLY.

Tags: i at the start of forward of step i, -1 at the start of the optimizer
step, i+1 when it ends.  Once a failure is known, every normal rank must
report after the failure was detected; then all equal tags T >= 0 mean
"stop now, resume at T", any -1 means "wait" (optimizer step in progress),
anything else is inconsistent with the barrier before the optimizer step.
No live rank in some data-parallel group means no replica: checkpoint.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass
class Cluster:
    n_ranks: int
    groups: list
    timeout: float
    created: float
    tag: dict = field(default_factory=dict)        # rank -> last tag
    seen: dict = field(default_factory=dict)       # rank -> time of last heartbeat
    reported: dict = field(default_factory=dict)   # rank -> time of failure report

    def heartbeat(self, r, tag, now):
        self.tag[r] = tag
        self.seen[r] = now

    def report_failure(self, r, now):
        self.reported.setdefault(r, now)

    def _last(self, r):
        return self.seen.get(r, self.created)

    def failed(self, now):
        return [r for r in range(self.n_ranks)
                if r in self.reported or now - self._last(r) > self.timeout]

    def decide(self, now):
        failed = set(self.failed(now))
        if not failed:
            return "continue", -1
        for g in set(self.groups):
            if all(r in failed for r in range(self.n_ranks) if self.groups[r] == g):
                return "checkpoint_fallback", -1
        detected = max(min(self.reported.get(r, float("inf")), self._last(r) + self.timeout) for r in failed)
        normal = [r for r in range(self.n_ranks) if r not in failed]
        fresh = [r in self.seen and self.seen[r] >= detected for r in normal]
        if not all(fresh) or any(self.tag[r] == -1 for r in normal):
            return "wait", -1
        tags = {self.tag[r] for r in normal}
        if len(tags) == 1:
            return "stop_and_restore", tags.pop()
        return "inconsistent", -1

    def donors(self, now):
        failed = set(self.failed(now))
        out = [-1] * self.n_ranks
        used = {}
        for r in range(self.n_ranks):
            if r not in failed:
                continue
            live = [q for q in range(self.n_ranks) if self.groups[q] == self.groups[r] and q not in failed]
            if live:
                k = used.get(self.groups[r], 0)
                out[r] = live[k % len(live)]
                used[self.groups[r]] = k + 1
        return out
