"""Coordinator behaviour on the host-simulated device (FAKE backend, no GPU).

Checks, for every policy: each request completes exactly once; critical ops are
never sharded; normal shards partition each op's tile space in tree-head order;
no normal shard sized next to a critical kernel exceeds the Eq. (2) grid limit;
one stream is FIFO; SEQUENTIAL never overlaps requests; deadlines, timed
release, draining shutdown and busy-object errors behave as documented.
"""
import ctypes
import time

import pytest

FAKE = 0x100000


@pytest.fixture(scope="module")
def L():
    from paper_2307_04339_amd import _lib
    _lib.load()
    return _lib


def _op(L, kind, **kw):
    d = L.OpDesc()
    d.kind = kind
    d.dtype = L.F16
    d.x = FAKE
    d.wt = FAKE
    d.y = FAKE
    for k, v in kw.items():
        setattr(d, k, v)
    h = ctypes.c_void_p()
    assert L.load().miriam_op_create(ctypes.byref(d), ctypes.byref(h)) == 0, L.load().miriam_last_error()
    return h


class _H:  # minimal op holder accepted by Coordinator.task
    def __init__(self, h):
        self.handle = h


def _net(L, sizes):
    """A chain of GEMM ops with the given tile counts (64x64 tiles)."""
    ops = []
    for t in sizes:
        ops.append(_H(_op(L, L.OP_GEMM, m=64 * t, nn=64, kk=64, tile=2)))
    return ops


def _coord(**kw):
    from paper_2307_04339_amd.runtime import Coordinator
    base = dict(backend="fake", log_launches=1, fake_n_cu=8, fake_slots_per_cu=2,
                fake_tile_ns=2000.0, fake_launch_ns=3000.0, quantum_us=10.0, profile_reps=1)
    base.update(kw)
    return Coordinator(**base)


def _collect(co, n, timeout=20.0):
    got = []
    t0 = time.time()
    while len(got) < n and time.time() - t0 < timeout:
        got.extend(co.poll())
        time.sleep(0.002)
    return got


@pytest.mark.parametrize("policy,segments,event_us", [("elastic", 0, 0.0), ("elastic", 1, 0.0), ("elastic", 1, 25.0),
                                                      ("elastic", 0, 1e9), ("sequential", 0, 0.0),
                                                      ("multistream", 0, 0.0), ("ib", 0, 0.0)])
def test_every_request_completes_once(L, policy, segments, event_us):
    # event_us: normal launches carry a completion event only every event_us of estimated work
    # (1e9: only each request's last launch)
    co = _coord(policy=policy, n_be_streams=2, inflight_depth=2, segments=segments, event_us=event_us)
    try:
        crit = co.task(_net(L, [3, 5, 2]))
        be1 = co.task(_net(L, [40, 17, 64] + [2] * 6 + [40]))
        be2 = co.task(_net(L, [9, 33]))
        tickets = []
        now = co.now_ns()
        for i in range(6):
            tickets.append(co.submit(crit, True, release_ns=now + i * 300_000))
        for i in range(5):
            tickets.append(co.submit(be1, False))
            tickets.append(co.submit(be2, False))
        recs = _collect(co, len(tickets))
        assert sorted(r.ticket for r in recs) == sorted(tickets)
        assert all(r.status == 0 for r in recs)
        assert all(r.t_end_ns >= r.t_start_ns >= r.t_release_ns > 0 for r in recs)
        co.drain(5000)
        assert co.poll() == []
        log = co.launch_log()
        st = co.stats()
        assert st.completed == len(tickets)
        assert st.eq2_violations == 0
        assert st.launches == len(log)
        # short ops (5 us each on the simulated device, quantum 10 us) run as captured pairs
        assert (st.segment_launches > 0) == (segments == 1)
        _check_log(log, policy)
    finally:
        co.shutdown()


@pytest.mark.parametrize("policy", ["elastic", "sequential"])
def test_submit_returns_the_ticket_of_its_request(L, policy):
    # Requests that finish while submit is still returning (tiny ops, a fast simulated device,
    # a submitting thread that can be descheduled) must still report their own ticket: the
    # dispatcher owns and frees a request once it is queued.
    co = _coord(policy=policy, n_be_streams=1, fake_tile_ns=1.0, fake_launch_ns=1.0, profile_reps=0)
    try:
        be = co.task(_net(L, [1]))
        tickets = [co.submit(be, False) for _ in range(3000)]
        recs = _collect(co, len(tickets), timeout=60.0)
        assert len(set(tickets)) == len(tickets)
        assert sorted(r.ticket for r in recs) == sorted(tickets)
    finally:
        co.shutdown()


def _check_log(log, policy):
    by_req = {}
    for r in log:
        by_req.setdefault((r.ticket, r.op_index), []).append(r)
        if r.criticality == 1 or policy != "elastic":
            # critical ops (and baselines) are never sharded
            assert (r.shard_begin, r.shard_len, r.grid, r.block) == (0, r.num_tiles, r.num_tiles, 256)
        if r.criticality == 0 and r.crit_busy:
            assert r.eq2_grid_limit > 0 and r.grid <= r.eq2_grid_limit
        assert 1 <= r.grid <= r.shard_len
    for (tk, oi), shards in by_req.items():
        # shards of one op: issued in increasing tile order, covering [0, T) exactly once
        cur = 0
        for s in shards:
            assert s.shard_begin == cur
            cur += s.shard_len
        assert cur == shards[0].num_tiles
    if policy != "sequential":
        for r in log:
            assert (r.stream == 0) == (r.criticality == 1)


def test_elastic_shards_follow_the_tree_and_eq2(L):
    from oracle import oracle as orc
    co = _coord(policy="elastic", n_be_streams=1, inflight_depth=1, quantum_us=6.0)
    try:
        crit = co.task(_net(L, [3] * 12))
        be = co.task(_net(L, [400, 256]))
        now = co.now_ns()
        tickets = [co.submit(be, False) for _ in range(12)]
        tickets += [co.submit(crit, True, release_ns=now + 200_000 + i * 700_000) for i in range(4)]
        recs = _collect(co, len(tickets))
        assert len(recs) == len(tickets)
        log = co.launch_log()
        normal = [r for r in log if r.criticality == 0]
        assert any(r.crit_busy for r in normal), "no shard was sized next to a critical kernel"
        assert any(r.shard_len < r.num_tiles for r in normal), "nothing was sharded"
        for r in normal:
            # each shard is a node of the op's shaded binary tree, taken at its head
            ln, _ = orc.tree_head(r.num_tiles, r.shard_begin, r.shard_len)
            assert ln == r.shard_len
            if r.crit_busy:
                # Eq. (2): 8 simulated CUs, critical kernels of 3 tiles -> 8 - 3 = 5
                assert r.eq2_grid_limit == orc.eq2_grid_limit(8, 3)
                assert r.grid <= r.eq2_grid_limit
    finally:
        co.shutdown()


def test_ib_kernels_advance_in_barrier_groups(L):
    # Two normal tasks of three kernels each, one long (64 tiles: 4 waves on the simulated
    # 8 x 2 slots) and one short (1 tile).  Under IB the short task's kernel k+1 waits for the
    # long task's kernel k, so it ends after two long kernels; on separate streams without
    # barriers it ends after its own three.
    tile_ns = 200_000.0
    long_ns = 4 * tile_ns
    lat = {}
    for policy in ("ib", "multistream"):
        co = _coord(policy=policy, n_be_streams=2, fake_tile_ns=tile_ns, fake_launch_ns=1000.0, profile_reps=0)
        try:
            ta = co.task(_net(L, [64, 64, 64]))
            tb = co.task(_net(L, [1, 1, 1]))
            # one common timed release, so both requests are released in the same dispatcher pass
            rel = co.now_ns() + 3_000_000
            ka = co.submit(ta, False, release_ns=rel)
            kb = co.submit(tb, False, release_ns=rel)
            recs = {r.ticket: r for r in _collect(co, 2)}
            assert set(recs) == {ka, kb} and all(r.status == 0 for r in recs.values())
            lat[policy] = recs[kb].t_end_ns - recs[kb].t_release_ns
            st = co.stats()
            assert st.barrier_groups == (3 if policy == "ib" else 0)
            log = co.launch_log()
            assert len(log) == 6
            for r in log:
                assert (r.shard_begin, r.shard_len, r.grid, r.block) == (0, r.num_tiles, r.num_tiles, 256)
            if policy == "ib":
                # one kernel per task per group, issued in op order: A0 B0 | A1 B1 | A2 B2
                by_issue = sorted(log, key=lambda r: r.t_issue_ns)
                assert [r.op_index for r in by_issue] == [0, 0, 1, 1, 2, 2]
        finally:
            co.shutdown()
    assert lat["ib"] >= 2 * long_ns
    assert lat["multistream"] < 2 * long_ns


def test_sequential_never_overlaps(L):
    co = _coord(policy="sequential", n_be_streams=2)
    try:
        crit = co.task(_net(L, [4, 4]))
        be = co.task(_net(L, [30, 30]))
        now = co.now_ns()
        tk = [co.submit(be, False) for _ in range(4)]
        tk += [co.submit(crit, True, release_ns=now + i * 150_000) for i in range(4)]
        recs = sorted(_collect(co, len(tk)), key=lambda r: r.t_start_ns)
        assert len(recs) == len(tk)
        for a, b in zip(recs, recs[1:]):
            assert a.t_end_ns <= b.t_start_ns
        assert all(r.stream == 0 for r in co.launch_log())
    finally:
        co.shutdown()


def test_fifo_within_a_task_and_critical_edf(L):
    co = _coord(policy="elastic", n_be_streams=1)
    try:
        be = co.task(_net(L, [20]))
        crit = co.task(_net(L, [2]))
        tks = [co.submit(be, False) for _ in range(5)]
        rel = co.now_ns() + 2_000_000
        late = co.submit(crit, True, release_ns=rel, deadline_ns=rel + 10**9)
        early = co.submit(crit, True, release_ns=rel, deadline_ns=rel + 10**6)
        recs = _collect(co, 7)
        normal = [r.ticket for r in sorted(recs, key=lambda r: r.t_end_ns) if r.criticality == 0]
        assert normal == tks
        first_crit = [r.ticket for r in co.launch_log() if r.criticality == 1][0]
        assert first_crit == early and late != early
    finally:
        co.shutdown()


def test_deadlines_and_timed_release(L):
    co = _coord()
    try:
        t = co.task(_net(L, [2]))
        now = co.now_ns()
        a = co.submit(t, True, release_ns=now + 3_000_000, deadline_ns=now + 10**10)
        b = co.submit(t, True, deadline_ns=now + 1)  # already missed
        recs = {r.ticket: r for r in _collect(co, 2)}
        assert recs[a].deadline_met == 1 and recs[b].deadline_met == 0
        assert recs[a].t_start_ns >= now + 3_000_000
    finally:
        co.shutdown()


def test_busy_objects_and_state_errors(L):
    lib = L.load()
    co = _coord()
    try:
        ops = _net(L, [50, 50])
        t = co.task(ops)
        now = co.now_ns()
        co.submit(t, False, release_ns=now + 50_000_000)  # held back 50 ms
        assert lib.miriam_task_destroy(t.handle) == L.EBUSY
        assert lib.miriam_op_destroy(ops[0].handle) == L.EBUSY
        assert lib.miriam_init(ctypes.byref(co.cfg)) == L.ESTATE
        assert lib.miriam_submit(None, 0, 0, 0, None) == L.EINVAL
        assert lib.miriam_submit(t.handle, 2, 0, 0, None) == L.EINVAL
        assert lib.miriam_drain(1) == L.EBUSY
    finally:
        co.shutdown()  # drains the held-back request first
    assert lib.miriam_poll((L.Completion * 1)(), 1) == L.ESTATE
    assert lib.miriam_op_destroy(ops[0].handle) == 0


def test_bad_configs_rejected(L):
    from paper_2307_04339_amd.runtime import default_config
    lib = L.load()
    for bad in [dict(policy=5), dict(n_be_streams=0), dict(n_be_streams=9), dict(inflight_depth=0),
                dict(top_frac=0.0), dict(quantum_us=0.0), dict(backend=3), dict(graphs=2), dict(graphs=-1),
                dict(busy_policy=3), dict(be_cu_reserve=-1), dict(policy=4), dict(crit_cu_exclusive=2),
                dict(crit_cu_exclusive=-1)]:
        c = default_config(**dict(dict(backend="fake"), **bad))
        assert lib.miriam_init(ctypes.byref(c)) == L.EINVAL, bad


@pytest.mark.parametrize("guard,warm", [(0, 0), (1, 0), (1, 1)])
def test_release_guard_keeps_normal_work_clear_of_timed_releases(L, guard, warm):
    co = _coord(release_guard=guard, warm_critical=warm, busy_policy=1, inflight_depth=4, quantum_us=100.0)
    try:
        be = co.task(_net(L, [20000, 20000]))
        cr = co.task(_net(L, [4]))
        now = co.now_ns()
        rels = [now + 4_000_000 + k * 2_000_000 for k in range(3)]
        for _ in range(3):
            co.submit(be, False)
        tks = [co.submit(cr, True, release_ns=r) for r in rels]
        got = {r.ticket: r for r in _collect(co, 6)}
        assert len(got) == 6 and all(r.status == 0 for r in got.values())
        log = [r for r in co.launch_log() if r.criticality == 0]
        assert log
        late = 0
        for rel in rels:
            before = [r for r in log if r.t_issue_ns < rel]
            assert before  # normal work runs up to each release
            # a shard issued before a release is estimated to end by it (launch and logging slack)
            late += sum(1 for r in before if r.t_issue_ns + 1000.0 * r.est_us > rel + 20_000)
        if guard:
            assert late == 0
        for tk, rel in zip(tks, rels):
            assert got[tk].t_start_ns >= rel
        # one warming pass ahead of each release that found normal work running
        assert co.stats().warm_launches == (len(rels) if warm else 0)
    finally:
        co.shutdown()


def test_armed_critical_requests_start_at_release(L):
    """Timed critical requests armed ahead of their release (kernels queued behind a gate)
    still start no earlier than the release, and critical work released while a gate is
    closed completes after it."""
    co = _coord(arm_lead_us=500.0, release_guard=1, busy_policy=1)
    try:
        be = co.task(_net(L, [2000, 2000]))
        cr = co.task(_net(L, [4, 4]))
        now = co.now_ns()
        rels = [now + 3_000_000 + k * 1_500_000 for k in range(4)]
        tks = [co.submit(cr, True, release_ns=r) for r in rels]
        for _ in range(4):
            co.submit(be, False)
        got = {r.ticket: r for r in _collect(co, 8)}
        assert len(got) == 8 and all(r.status == 0 for r in got.values())
        for tk, rel in zip(tks, rels):
            assert got[tk].t_start_ns >= rel and got[tk].t_end_ns >= rel
        assert co.stats().armed_releases == len(rels)
        # an immediate critical request while the next one is armed
        rel = co.now_ns() + 2_000_000
        a = co.submit(cr, True, release_ns=rel)
        while co.stats().armed_releases < len(rels) + 1:
            time.sleep(0.0001)
        b = co.submit(cr, True)
        got = {r.ticket: r for r in _collect(co, 2)}
        assert got[a].status == 0 and got[b].status == 0
        assert got[a].t_start_ns >= rel
    finally:
        co.shutdown()


def test_whole_requests_launch_only_clear_of_timed_releases(L):
    # whole_when_clear: a normal request goes out as one whole-request launch only while no
    # critical work is pending or running and it is estimated to end before the next timed
    # release; near a release its ops are sharded (and held by the guard) as usual
    co = _coord(release_guard=1, whole_when_clear=1, busy_policy=1, inflight_depth=4, quantum_us=100.0,
                fake_tile_ns=2000.0, fake_launch_ns=3000.0)
    try:
        crit = co.task(_net(L, [4, 4]))
        be = co.task(_net(L, [32, 32, 32]))
        now = co.now_ns()
        period = 2_000_000
        rel = [now + 3_000_000 + i * period for i in range(5)]
        tk = [co.submit(crit, True, release_ns=r) for r in rel]
        tk += [co.submit(be, False) for _ in range(30)]
        recs = _collect(co, len(tk), timeout=30.0)
        assert sorted(r.ticket for r in recs) == sorted(tk) and all(r.status == 0 for r in recs)
        st = co.stats()
        assert st.whole_clear_launches > 0
        log = co.launch_log()
        crit_t = {r.ticket for r in recs if r.criticality == 1}
        # every whole normal request was issued with its estimated end before the next release
        whole = {}
        for r in log:
            if r.criticality == 0:
                whole.setdefault(r.ticket, []).append(r)
        # a whole launch logs each op at its full grid (32 tiles); shards sized by the
        # coordinator use at most the simulated 8 x 2 workgroup slots
        def is_whole(rs):
            return len(rs) == 3 and all(x.shard_len == x.num_tiles == x.grid for x in rs)
        assert sum(1 for rs in whole.values() if is_whole(rs)) == st.whole_clear_launches
        for rs in whole.values():
            if is_whole(rs):
                t_issue = rs[0].t_issue_ns
                est_end = t_issue + int(1000 * sum(x.est_us for x in rs))
                nxt = [r for r in rel if r > t_issue]
                assert not nxt or est_end <= nxt[0]
        assert crit_t
    finally:
        co.shutdown()


@pytest.mark.parametrize("policy,fail_at", [("elastic", 5), ("elastic", 1), ("sequential", 3),
                                            ("multistream", 2), ("ib", 4)])
def test_injected_launch_failure_ends_one_request(L, policy, fail_at):
    # the simulated device fails its fail_at-th launch: exactly the request that launch belonged
    # to completes with MIRIAM_EHIP, the counters of its task's ops are cleared once per op, and
    # every other request, including ones submitted after the failure, completes normally
    co = _coord(policy=policy, n_be_streams=2, inflight_depth=2, fake_fail_launch=fail_at, profile_reps=0)
    try:
        crit = co.task(_net(L, [3, 5, 2]))
        be = co.task(_net(L, [9, 17, 4, 6]))
        tickets = [co.submit(crit, True)]
        tickets += [co.submit(be, False) for _ in range(3)]
        recs = _collect(co, len(tickets))
        assert sorted(r.ticket for r in recs) == sorted(tickets)
        bad = [r for r in recs if r.status != 0]
        assert len(bad) == 1
        assert bad[0].status == -3
        st = co.stats()
        assert st.failed_requests == 1
        n_ops = 3 if bad[0].criticality == 1 else 4
        assert st.failed_pass_resets == n_ops
        later = [co.submit(be, False), co.submit(crit, True)]
        recs2 = _collect(co, 2)
        assert sorted(r.ticket for r in recs2) == sorted(later)
        assert all(r.status == 0 for r in recs2)
        assert co.stats().failed_requests == 1
    finally:
        co.shutdown()
