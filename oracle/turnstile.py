"""Plain model of the segment turnstile's controller (Sections 4.2-4.3).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path never
imports, calls or links it, and it imports nothing from the product package.

What the paper fixes (Section 4.2, "Rank-Aligned Segment Boundaries", and
Section 4.3, the turnstile step and its rendezvous):

* a P epoch e publishes safe boundary ids i = 0, 1, ... in increasing order,
  from exactly one producer;
* the controller holds r, the largest boundary reached (-1 at the start of
  an epoch), the permitted endpoint p, a positive span K and the task state;
* p starts at 0 when a ready D has not been enqueued yet (D is ordered before
  P's first GPU work) and at K when D is already enqueued;
* P: while p = 0 it waits before any GPU work; after publishing i it waits
  while i >= p (so it stops at i = p); after its final segment it reports
  TaskDone;
* D: if p > 0 it waits until r >= p or TaskDone (p = 0 needs no
  publication), enqueues its iteration, then an active task gets
  p <- p + K; completed tasks take no new permit;
* refused: stale or duplicate epochs, publications without a producer,
  boundaries that do not increase, boundaries beyond the current permit.

Readings where the text leaves a choice (listed with the other readings of
the paper in the design notes): a publication while p = 0 is beyond the
permit (P may not have started); a new epoch may not begin while the
previous one is still active; D may not release without having entered, nor
enter twice; an epoch may end (TaskDone) at any boundary; a D iteration that
entered before the epoch began (the D that "already enqueued" refers to)
releases no permit of that epoch.

Waits are modelled without blocking: ``wait_*`` answers "ok" when the wait
would pass now and "wait" when it would block, changing nothing then.
Results are the strings "ok", "wait", "rejected" and "invalid".
"""

from __future__ import annotations

IDLE, ACTIVE, DONE = "idle", "active", "done"


class Turnstile:
    def __init__(self, span: int):
        if span < 1:
            raise ValueError("span must be positive")
        self.K = span
        self.highest = -1      # highest epoch ever begun
        self.e = -1            # current epoch
        self.r = -1            # largest published boundary of the epoch
        self.p = 0             # permitted endpoint
        self.task = IDLE
        self.d_inside = False
        self.d_entry_epoch = None  # epoch active when D entered, if any
        self.rounds = 0        # releases that advanced an active task's permit
        self.rejected = 0
        self.events = []       # accepted transitions: (kind, epoch, value)

    # -- helpers
    def _reject(self):
        self.rejected += 1
        return "rejected"

    def _active(self, e):
        return self.task == ACTIVE and e == self.e

    def state(self):
        return dict(epoch=self.e, reached=self.r, permit=self.p, span=self.K, task=self.task,
                    rounds=self.rounds, rejected=self.rejected)

    # -- policy
    def set_span(self, span):
        if span < 1:
            return "invalid"
        self.K = span
        return "ok"

    # -- P side
    def begin(self, e, d_enqueued):
        if e <= self.highest or self.task == ACTIVE:
            return self._reject()
        self.highest = self.e = e
        self.r = -1
        self.p = self.K if d_enqueued else 0
        self.task = ACTIVE
        self.rounds = 0
        self.events.append(("begin", e, self.p))
        return "ok"

    def publish(self, e, i):
        if i < 0:
            return "invalid"
        if not self._active(e):
            return self._reject()          # no producer registered for e
        if i <= self.r:
            return self._reject()          # not increasing (duplicates included)
        if self.p == 0 or i > self.p:
            return self._reject()          # beyond the permit
        self.r = i
        self.events.append(("publish", e, i))
        return "ok"

    def wait_permit(self, e, i):
        """i = -1: the wait before P's first GPU work; otherwise the wait after
        publishing i."""
        if i < -1:
            return "invalid"
        if not self._active(e) or (i >= 0 and i != self.r):
            return self._reject()
        passes = self.p > 0 if i < 0 else i < self.p
        if not passes:
            return "wait"
        self.events.append(("resume", e, i))
        return "ok"

    def done(self, e):
        if not self._active(e):
            return self._reject()
        self.task = DONE
        self.events.append(("done", e, self.r))
        return "ok"

    # -- D side
    def wait_boundary(self):
        if self.d_inside:
            return self._reject()
        if self.task == ACTIVE and self.p > 0 and self.r < self.p:
            return "wait"
        self.d_inside = True
        self.d_entry_epoch = self.e if self.task == ACTIVE else None
        self.events.append(("enter", self.e, self.p))
        return "ok"

    def release(self):
        if not self.d_inside:
            return self._reject()
        self.d_inside = False
        if self.task == ACTIVE and self.d_entry_epoch == self.e:
            self.p += self.K
            self.rounds += 1
        self.events.append(("release", self.e, self.p))
        return "ok"


def interior_stops(boundaries: int, span: int) -> int:
    """Number of D releases an epoch of `boundaries` boundaries (ids
    0..boundaries-1) needs when it starts with p = K: P stops at every
    p = K, 2K, ... that it reaches before its last boundary."""
    return (boundaries - 1) // span


def check_log(events, span):
    """Check a sequence of logged transitions (kind, epoch, value) of one
    epoch against the protocol by replaying it through the model, then
    check the ordering property of Section 4.3: for every D entry at an
    endpoint p > 0 of an active task, P published p before the entry and P
    resumed past p only after the following release.  Returns a list of
    problems (empty when the log is valid)."""
    problems = []
    t = Turnstile(span)
    for n, (kind, e, v) in enumerate(events):
        if kind == "begin":
            res = t.begin(e, v > 0)
            if res == "ok" and t.p != v:
                problems.append(f"event {n}: begin gives p={t.p}, log says {v}")
        elif kind == "publish":
            res = t.publish(e, v)
        elif kind == "resume":
            res = t.wait_permit(e, v)
        elif kind == "done":
            res = t.done(e)
        elif kind == "enter":
            res = t.wait_boundary()
            if res == "ok" and t.p != v:
                problems.append(f"event {n}: enter at p={t.p}, log says {v}")
        elif kind == "release":
            res = t.release()
            if res == "ok" and t.p != v:
                problems.append(f"event {n}: release gives p={t.p}, log says {v}")
        else:
            res = "unknown kind"
        if res != "ok":
            problems.append(f"event {n} {kind, e, v}: {res}")
    # ordering: publish(p) < enter(p) < release < resume(p)
    pos = {}
    for n, (kind, e, v) in enumerate(events):
        pos.setdefault((kind, e, v), n)
    for n, (kind, e, v) in enumerate(events):
        if kind != "enter" or v <= 0:
            continue
        done_before = any(k == "done" and ee == e for k, ee, _ in events[:n])
        if done_before:
            continue
        pub = pos.get(("publish", e, v))
        if pub is None or pub > n:
            problems.append(f"event {n}: D entered at p={v} before P published it")
        rel = next((m for m in range(n + 1, len(events)) if events[m][0] == "release"), None)
        res = pos.get(("resume", e, v))
        if res is not None and (rel is None or res < rel):
            problems.append(f"event {n}: P resumed past {v} before D released")
    return problems
