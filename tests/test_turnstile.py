"""Segment turnstile (Sections 4.2-4.3): the oracle model pinned to the
protocol's stated rules and properties, then the native controller checked
against the model operation by operation, and its blocking waits with real
threads.  Host only: no GPU is touched."""

import copy
import random
import threading
import time

import pytest

from oracle import turnstile as O

# ---------------------------------------------------------------- oracle pins


def test_ready_d_goes_before_p_enters_the_gpu():
    # p = 0: P waits before any GPU work; D needs no publication; its release
    # gives p = K and lets P start.
    t = O.Turnstile(2)
    assert t.begin(0, d_enqueued=False) == "ok" and t.p == 0
    assert t.wait_permit(0, -1) == "wait"
    assert t.publish(0, 0) == "rejected"  # P may not have started
    assert t.wait_boundary() == "ok"
    assert t.release() == "ok" and t.p == 2
    assert t.wait_permit(0, -1) == "ok"


def test_enqueued_d_lets_p_start_with_k():
    t = O.Turnstile(3)
    assert t.begin(0, d_enqueued=True) == "ok" and t.p == 3
    assert t.wait_permit(0, -1) == "ok"


def test_p_stops_at_the_permitted_endpoint():
    t = O.Turnstile(2)
    t.begin(0, True)
    for i in range(2):
        assert t.publish(0, i) == "ok"
        assert t.wait_permit(0, i) == "ok"  # i < p
    assert t.publish(0, 2) == "ok"
    assert t.wait_permit(0, 2) == "wait"  # i = p: stop
    assert t.publish(0, 3) == "rejected"  # beyond the permit


def test_d_waits_for_the_endpoint_or_taskdone():
    t = O.Turnstile(2)
    t.begin(0, True)
    t.publish(0, 0)
    t.publish(0, 1)
    assert t.wait_boundary() == "wait"  # r = 1 < p = 2
    t.publish(0, 2)
    assert t.wait_boundary() == "ok"
    assert t.release() == "ok" and t.p == 4 and t.rounds == 1
    t.publish(0, 3)
    assert t.wait_boundary() == "wait"
    assert t.done(0) == "ok"  # TaskDone before the endpoint
    assert t.wait_boundary() == "ok"
    assert t.release() == "ok" and t.p == 4 and t.rounds == 1  # completed: no new permit


def test_rejections():
    t = O.Turnstile(2)
    assert t.publish(0, 0) == "rejected"  # no producer registered
    assert t.done(0) == "rejected"
    assert t.begin(5, True) == "ok"
    assert t.begin(6, True) == "rejected"  # previous epoch still active
    assert t.publish(4, 0) == "rejected"  # stale epoch
    assert t.publish(5, 0) == "ok"
    assert t.publish(5, 0) == "rejected"  # duplicate boundary
    assert t.publish(5, 2) == "ok"  # increasing, within the permit
    assert t.publish(5, 1) == "rejected"  # not increasing
    assert t.wait_permit(5, 0) == "rejected"  # not the last published boundary
    assert t.done(5) == "ok"
    assert t.publish(5, 3) == "rejected"  # producer gone
    assert t.begin(5, True) == "rejected"  # duplicate epoch
    assert t.begin(3, True) == "rejected"  # stale epoch
    assert t.release() == "rejected"  # D not inside
    assert t.wait_boundary() == "ok"
    assert t.wait_boundary() == "rejected"  # already inside
    assert t.rejected == 12
    assert t.publish(6, -1) == "invalid" and t.set_span(0) == "invalid"
    assert t.rejected == 12


def test_global_enqueue_epoch_takes_one_rendezvous():
    # Section 7.4 (ordering ladder): each Global-Enqueue epoch passes one
    # rendezvous after its 40 dispatch boundaries: with K >= 40 P never stops
    # inside the epoch and D's only entry comes after TaskDone.
    assert O.interior_stops(40, 40) == 0 and O.interior_stops(40, 1000) == 0
    t = O.Turnstile(40)
    t.begin(0, True)
    for i in range(40):
        assert t.publish(0, i) == "ok"
        if i < 39:
            assert t.wait_boundary() == "wait"
        assert t.wait_permit(0, i) == "ok"
    assert t.done(0) == "ok"
    assert t.wait_boundary() == "ok" and t.release() == "ok"
    assert t.rounds == 0


def _explore(B, K, d_enqueued, d_budget):
    """Every interleaving of one P epoch's program (wait before the GPU, then
    publish i / wait i for i < B, then TaskDone) with a D thread that enters
    and releases up to d_budget times.  Yields (events, model) of every
    complete run; raises on an invariant violation or a deadlock."""
    P = [("begin",), ("wait", -1)] + [s for i in range(B) for s in (("publish", i), ("wait", i))] + [("done",)]

    def step_p(t, pc):
        op = P[pc]
        if op[0] == "begin":
            return t.begin(0, d_enqueued)
        if op[0] == "wait":
            return t.wait_permit(0, op[1])
        if op[0] == "publish":
            return t.publish(0, op[1])
        return t.done(0)

    stack = [(O.Turnstile(K), 0, 0, False)]  # model, P pc, D entries, D inside
    while stack:
        t, pc, nd, inside = stack.pop()
        # invariants of every reachable state
        if t.task == O.ACTIVE and t.p > 0:
            assert t.r <= t.p
        moved = False
        if pc < len(P):
            u = copy.deepcopy(t)
            res = step_p(u, pc)
            assert res in ("ok", "wait"), (P[pc], res)
            if res == "ok":
                moved = True
                stack.append((u, pc + 1, nd, inside))
        if inside:
            u = copy.deepcopy(t)
            assert u.release() == "ok"
            moved = True
            stack.append((u, pc, nd, False))
        elif nd < d_budget:
            u = copy.deepcopy(t)
            res = u.wait_boundary()
            if res == "ok":
                if u.task == O.ACTIVE and u.p > 0:
                    assert u.r == u.p  # D enters exactly at the endpoint
                moved = True
                stack.append((u, pc, nd + 1, True))
        if pc == len(P) and not inside:
            yield t
            continue
        if not moved:
            # P blocked at a permit wait: only acceptable when D has no budget left
            assert nd == d_budget, f"deadlock at pc={pc} state={t.state()}"


@pytest.mark.parametrize("B", [1, 2, 3, 5])
@pytest.mark.parametrize("K", [1, 2, 3])
@pytest.mark.parametrize("d_enqueued", [True, False])
def test_every_interleaving_keeps_the_protocol(B, K, d_enqueued):
    need = O.interior_stops(B, K) + (0 if d_enqueued else 1)
    runs = 0
    for t in _explore(B, K, d_enqueued, d_budget=need + 2):
        runs += 1
        assert t.rounds == need
        assert O.check_log(t.events, K) == []
        # boundaries published per segment: K + 1 in the first (0..K), then K
        # (a segment ends at a release that moved the permit)
        seg, sizes, p = 0, [], 0
        for kind, _, v in t.events:
            if kind == "publish":
                seg += 1
            elif kind == "begin":
                p = v
            elif kind == "release" and v > p:
                p = v
                if seg:
                    sizes.append(seg)
                    seg = 0
        sizes.append(seg)
        assert sum(sizes) == B
        # (the last segment may publish nothing: P stopped at its final
        # boundary and only finishes that layer after the release)
        assert sizes[0] == min(B, K + 1) and all(s == K for s in sizes[1:-1])
        assert len(sizes) == 1 or 0 <= sizes[-1] <= K
    assert runs > 0


def test_check_log_catches_misordered_logs():
    t = O.Turnstile(1)
    t.begin(0, True)
    t.wait_permit(0, -1)
    t.publish(0, 0)
    t.publish(0, 1)
    t.wait_boundary()
    t.release()
    t.wait_permit(0, 1)
    good = list(t.events)
    assert O.check_log(good, 1) == []
    # D entering before P reached the endpoint
    bad = good[:3] + [good[4]] + [good[3]] + good[5:]
    assert O.check_log(bad, 1)
    # P resuming past the endpoint before D's release
    bad = good[:5] + [good[6], good[5]]
    assert O.check_log(bad, 1)
    # a different span than the one logged
    assert O.check_log(good, 2)


# ---------------------------------------------------------------- native controller

M = pytest.importorskip("paper_2609_00993_amd.moepd")

TASK = {M.MOE_TS_IDLE: O.IDLE, M.MOE_TS_ACTIVE: O.ACTIVE, M.MOE_TS_DONE: O.DONE}
RES = {M.MOE_OK: "ok", M.MOE_ERR_REJECTED: "rejected", M.MOE_ERR_TIMEOUT: "wait", M.MOE_ERR_INVALID_ARG: "invalid"}
KIND = {M.MOE_TS_EV_BEGIN: "begin", M.MOE_TS_EV_PUBLISH: "publish", M.MOE_TS_EV_RESUME: "resume",
        M.MOE_TS_EV_ENTER: "enter", M.MOE_TS_EV_RELEASE: "release", M.MOE_TS_EV_DONE: "done"}


@pytest.fixture
def native():
    made = []

    def make(span, log=0):
        st, ts = M.moe_turnstile_create(span, log)
        M.check(st)
        made.append(ts)
        return ts

    yield make
    for ts in made:
        M.moe_turnstile_destroy(ts)


def _state(ts):
    st, q = M.moe_turnstile_query(ts)
    M.check(st)
    return dict(epoch=q.epoch, reached=q.reached, permit=q.permit, span=q.span, task=TASK[q.task],
                rounds=q.rounds, rejected=q.rejected)


@pytest.mark.parametrize("seed", range(6))
def test_native_controller_matches_the_model(native, seed):
    rng = random.Random(seed)
    K = rng.randint(1, 3)
    ts, t = native(K), O.Turnstile(K)
    for n in range(3000):
        e = rng.choice([t.e - 1, t.e, t.e, t.e, t.highest + 1, t.highest + 2])
        op = rng.choices(["span", "begin", "publish", "permit", "done", "enter", "release"],
                         weights=[1, 3, 12, 10, 2, 8, 8])[0]
        if op == "span":
            k = rng.randint(0, 4)
            got, want = RES[M.moe_turnstile_set_span(ts, k)], t.set_span(k)
        elif op == "begin":
            d = rng.random() < 0.5
            got, want = RES[M.moe_turnstile_begin(ts, e, d)], t.begin(e, d)
        elif op == "publish":
            i = rng.choice([t.r + 1, t.r + 1, t.r + 2, t.r, t.p, t.p + 1, -1])
            got, want = RES[M.moe_turnstile_publish(ts, e, i)], t.publish(e, i)
        elif op == "permit":
            i = rng.choice([t.r, t.r, -1, t.r - 1, -2])
            got, want = RES[M.moe_turnstile_wait_permit(ts, e, i, 0)], t.wait_permit(e, i)
        elif op == "done":
            got, want = RES[M.moe_turnstile_done(ts, e)], t.done(e)
        elif op == "enter":
            got, want = RES[M.moe_turnstile_wait_boundary(ts, 0)], t.wait_boundary()
        else:
            got, want = RES[M.moe_turnstile_release(ts)], t.release()
        assert got == want, (n, op, e, t.state())
        assert _state(ts) == t.state(), (n, op)


def test_native_rejects_bad_arguments(native):
    ts = native(1)
    assert M.moe_turnstile_create(0, 0)[0] == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_create(1, -1)[0] == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_create(1, (1 << 20) + 1)[0] == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_set_span(None, 1) == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_begin(None, 0, True) == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_wait_boundary(ts, -1) == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_wait_permit(ts, 0, -1, -5) == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_release(None) == M.MOE_ERR_INVALID_ARG
    assert M.moe_turnstile_destroy(None) == M.MOE_OK
    assert M.moe_status_string(M.MOE_ERR_REJECTED) != "unknown status"
    assert M.moe_status_string(M.MOE_ERR_TIMEOUT) != "unknown status"
    assert _state(ts)["rejected"] == 0


def _later(fn, delay):
    th = threading.Timer(delay, fn)
    th.start()
    return th


def test_d_wait_is_woken_by_the_publication(native):
    ts = native(2)
    M.check(M.moe_turnstile_begin(ts, 0, True))
    for i in range(2):
        M.check(M.moe_turnstile_publish(ts, 0, i))
    th = _later(lambda: M.moe_turnstile_publish(ts, 0, 2), 0.05)
    t0 = time.perf_counter()
    assert M.moe_turnstile_wait_boundary(ts, 5_000_000) == M.MOE_OK
    waited = time.perf_counter() - t0
    th.join()
    assert 0.04 < waited < 2.0
    st, q = M.moe_turnstile_query(ts)
    assert q.d_wait_us > 30_000 and q.d_entries == 1


def test_p_wait_is_woken_by_the_release(native):
    ts = native(1)
    M.check(M.moe_turnstile_begin(ts, 0, True))
    M.check(M.moe_turnstile_publish(ts, 0, 0))
    M.check(M.moe_turnstile_publish(ts, 0, 1))
    M.check(M.moe_turnstile_wait_boundary(ts, 0))

    th = _later(lambda: M.moe_turnstile_release(ts), 0.05)
    t0 = time.perf_counter()
    assert M.moe_turnstile_wait_permit(ts, 0, 1, 5_000_000) == M.MOE_OK
    assert time.perf_counter() - t0 > 0.04
    th.join()


def test_waits_time_out_without_changing_state(native):
    ts = native(1)
    M.check(M.moe_turnstile_begin(ts, 0, False))
    before = _state(ts)
    t0 = time.perf_counter()
    assert M.moe_turnstile_wait_permit(ts, 0, -1, 30_000) == M.MOE_ERR_TIMEOUT
    assert time.perf_counter() - t0 >= 0.029
    M.check(M.moe_turnstile_wait_boundary(ts, 0))
    M.check(M.moe_turnstile_release(ts))
    M.check(M.moe_turnstile_wait_permit(ts, 0, -1, 0))
    M.check(M.moe_turnstile_publish(ts, 0, 0))
    M.check(M.moe_turnstile_publish(ts, 0, 1))
    assert M.moe_turnstile_wait_boundary(ts, 0) == M.MOE_OK
    assert M.moe_turnstile_wait_permit(ts, 0, 1, 20_000) == M.MOE_ERR_TIMEOUT
    assert _state(ts)["rejected"] == before["rejected"]


def _p_thread(ts, epoch, B, d_enqueued, errors):
    try:
        M.check(M.moe_turnstile_begin(ts, epoch, d_enqueued))
        M.check(M.moe_turnstile_wait_permit(ts, epoch, -1, 5_000_000))
        for i in range(B):
            M.check(M.moe_turnstile_publish(ts, epoch, i))
            M.check(M.moe_turnstile_wait_permit(ts, epoch, i, 5_000_000))
        M.check(M.moe_turnstile_done(ts, epoch))
    except Exception as exc:  # reported by the test body
        errors.append(exc)


@pytest.mark.parametrize("K,B", [(1, 5), (2, 7), (3, 3), (4, 9)])
def test_two_threads_follow_the_protocol(native, K, B):
    ts = native(K, log=4096)
    stop = threading.Event()
    errors = []

    def d_loop():
        while not stop.is_set():
            st = M.moe_turnstile_wait_boundary(ts, 2_000)
            if st == M.MOE_ERR_TIMEOUT:
                continue
            if st != M.MOE_OK:
                errors.append(st)
                return
            time.sleep(0.0002)  # the D iteration's enqueue
            M.check(M.moe_turnstile_release(ts))

    d = threading.Thread(target=d_loop)
    d.start()
    try:
        for epoch in range(3):
            _p_thread(ts, epoch, B, d_enqueued=epoch % 2 == 0, errors=errors)
            st, q = M.moe_turnstile_query(ts)
            assert q.task == M.MOE_TS_DONE
            assert q.rounds == O.interior_stops(B, K) + (0 if epoch % 2 == 0 else 1)
    finally:
        stop.set()
        d.join()
    assert not errors
    st, ev = M.moe_turnstile_log(ts, 4096)
    M.check(st)
    events = [(KIND[k], e, v) for k, e, v, _ in ev]
    for epoch in range(3):
        # D entries between epochs belong to no epoch; replay each epoch's own
        # transitions (those D entries that fall inside it included).
        first = events.index(("begin", epoch, K if epoch % 2 == 0 else 0))
        last = max(n for n, x in enumerate(events) if x[0] == "done" and x[1] == epoch)
        seg = events[first:last + 1]
        # a D inside at the epoch's start enters before it; drop an unmatched release
        if seg and any(x[0] == "release" for x in seg):
            opens = 0
            clean = []
            for x in seg:
                if x[0] == "enter":
                    opens += 1
                elif x[0] == "release":
                    if opens == 0:
                        continue
                    opens -= 1
                clean.append(x)
            seg = clean
        assert O.check_log(seg, K) == [], (epoch, seg)
    ts_ns = [t for *_, t in ev]
    assert ts_ns == sorted(ts_ns)
