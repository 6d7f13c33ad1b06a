"""The coordinator on the GPU: under every policy, with whole-request launches
replayed from captured HIP graphs or issued op by op, the networks' outputs are
bitwise identical to one eager forward pass, on every replay, with eager device
work between replays; a captured request is one launch that still accounts for
each of its ops, and normal shards sized next to it keep the Eq. (2) limit."""
import pytest
import torch

from gpu_util import bits, gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


def _nan_outputs(net):
    for l in net.layers:
        l.t["y"].fill_(float("nan"))


@pytest.mark.parametrize("policy,graphs,segments,event_us",
                         [(p, g, 0, 0.0) for p in ("elastic", "sequential", "multistream", "ib") for g in (0, 1)]
                         + [("elastic", 1, 1, 0.0), ("elastic", 1, 1, 30.0)])
def test_coordinator_outputs_match_eager(policy, graphs, segments, event_us):
    from paper_2307_04339_amd import models
    from paper_2307_04339_amd.runtime import Coordinator
    crit = models.resnet18(batch=1, dtype="f16")
    be = models.mobilenetv2(batch=4, dtype="bf16")
    for n in (crit, be):
        n.forward()
    torch.cuda.synchronize()
    ref = {n.name: [bits(l.t["y"]) for l in n.layers] for n in (crit, be)}
    co = Coordinator(policy=policy, graphs=graphs, segments=segments, event_us=event_us, profile_reps=1,
                     log_launches=1,
                     n_be_streams=1, inflight_depth=2, quantum_us=20.0)
    try:
        ct = co.task(crit.ops())
        bt = co.task(be.ops())
        reps = 3
        for rep in range(reps):
            _nan_outputs(crit)
            _nan_outputs(be)
            junk = torch.randn(1 << 20, device="cuda")
            float((junk * 2.0).sum())  # eager device work between replays
            torch.cuda.synchronize()
            tb = co.submit(bt, False)
            tc = co.submit(ct, True)
            tb2 = co.submit(bt, False)
            co.drain(60000)
            recs = {r.ticket: r for r in co.poll()}
            assert set(recs) == {tb, tc, tb2}
            assert all(r.status == 0 for r in recs.values())
            assert recs[tc].n_shards == len(crit.layers)
            torch.cuda.synchronize()
            for n in (crit, be):
                for l, r in zip(n.layers, ref[n.name]):
                    assert bits(l.t["y"]) == r, (policy, graphs, rep, n.name, l.name)
        st = co.stats()
        log = co.launch_log()
        crit_recs = [r for r in log if r.criticality == 1]
        assert len(crit_recs) == reps * len(crit.layers)
        assert all(r.shard_begin == 0 and r.shard_len == r.num_tiles and r.block == 256 for r in crit_recs)
        assert st.launches == len(log)
        assert st.eq2_violations == 0
        # requests launched whole (IB launches kernel by kernel, a barrier after each)
        whole = {"elastic": reps, "ib": 0}.get(policy, 3 * reps)
        assert st.graph_launches == (whole if graphs else 0)
        assert (st.barrier_groups > 0) == (policy == "ib")
        assert (st.segment_launches > 0) == (segments == 1)
    finally:
        co.shutdown()


@pytest.mark.parametrize("arm_lead_us,whole", [(0.0, 0), (500.0, 0), (500.0, 1)])
def test_warmed_periodic_critical_requests_match_eager(arm_lead_us, whole):
    """Timed critical releases with normal work running: the release guard holds normal
    shards and a cache-warming pass runs ahead of each release, and (arm_lead_us > 0) each
    critical request is queued behind a gate before its release; with whole_when_clear, normal
    requests that fit before the next release run as whole-request launches.  Outputs stay
    bitwise equal and armed requests complete after their release."""
    from paper_2307_04339_amd import models
    from paper_2307_04339_amd.runtime import Coordinator
    crit = models.resnet18(batch=1, dtype="f16")
    be = models.vgg16(batch=2, dtype="f16")
    for n in (crit, be):
        n.forward()
    torch.cuda.synchronize()
    ref = {n.name: [bits(l.t["y"]) for l in n.layers] for n in (crit, be)}
    co = Coordinator(policy="elastic", graphs=1, release_guard=1, warm_critical=1, busy_policy=1,
                     profile_reps=1, n_be_streams=1, inflight_depth=4, inflight_us=100.0, quantum_us=40.0,
                     arm_lead_us=arm_lead_us, whole_when_clear=whole)
    try:
        ct = co.task(crit.ops())
        bt = co.task(be.ops())
        for rep in range(2):
            _nan_outputs(crit)
            _nan_outputs(be)
            torch.cuda.synchronize()
            t0 = co.now_ns() + 2_000_000
            tks = [co.submit(ct, True, release_ns=t0 + k * 1_500_000) for k in range(4)]
            btk = [co.submit(bt, False) for _ in range(6)]
            co.drain(60000)
            recs = {r.ticket: r for r in co.poll()}
            assert set(recs) == set(tks) | set(btk)
            assert all(r.status == 0 for r in recs.values())
            for k, tk in enumerate(tks):
                assert recs[tk].t_start_ns >= t0 + k * 1_500_000
            torch.cuda.synchronize()
            for n in (crit, be):
                for l, r in zip(n.layers, ref[n.name]):
                    assert bits(l.t["y"]) == r, (rep, n.name, l.name)
        st = co.stats()
        assert st.warm_launches >= 1
        assert st.graph_launches == 8 + st.whole_clear_launches
        assert (st.whole_clear_launches > 0) == (whole == 1)
        assert st.armed_releases == (8 if arm_lead_us > 0 else 0)
    finally:
        co.shutdown()


@pytest.mark.parametrize("limit_us,open_after_us", [(300, -1), (50000, 1000), (2000, 0)])
def test_release_gate_ends_on_flag_or_limit(limit_us, open_after_us):
    """The gate that holds an armed critical request ends when the host raises its flag, and
    on its own wall-clock limit when the flag is never raised."""
    import ctypes
    from paper_2307_04339_amd import _lib as L
    lib = L.load()
    s = torch.cuda.Stream()
    held = ctypes.c_double()
    assert lib.miriam_gate_check(ctypes.c_void_p(s.cuda_stream), limit_us, open_after_us, ctypes.byref(held)) == 0, \
        lib.miriam_last_error()
    expect = limit_us if open_after_us < 0 else min(open_after_us, limit_us)
    assert held.value >= 0.8 * expect, (held.value, expect)
    assert held.value <= expect + 2000.0, (held.value, expect)
    # the stream runs normally afterwards
    with torch.cuda.stream(s):
        x = torch.ones(1024, device="cuda") * 2.0
    s.synchronize()
    assert float(x.sum()) == 2048.0


@pytest.mark.parametrize("policy,crit_excl", [("multistream", 0), ("elastic", 0), ("elastic", 1)])
def test_cu_masked_normal_streams_match_eager(policy, crit_excl):
    """Normal streams created with a compute-unit mask (64 CUs left to the critical stream, which
    with crit_excl has only those): every request completes with outputs bitwise equal to the
    eager forward pass, and a reserve of every CU is rejected."""
    from paper_2307_04339_amd import models
    from paper_2307_04339_amd import _lib as L
    from paper_2307_04339_amd.runtime import Coordinator
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    with pytest.raises(L.MiriamError):
        Coordinator(policy=policy, be_cu_reserve=n_cu, profile_reps=1)
    crit = models.resnet18(batch=1, dtype="f16")
    be = models.mobilenetv2(batch=4, dtype="bf16")
    for n in (crit, be):
        n.forward()
    torch.cuda.synchronize()
    ref = {n.name: [bits(l.t["y"]) for l in n.layers] for n in (crit, be)}
    co = Coordinator(policy=policy, be_cu_reserve=64, profile_reps=1, n_be_streams=1, inflight_depth=2,
                     quantum_us=20.0, crit_cu_exclusive=crit_excl)
    try:
        ct = co.task(crit.ops())
        bt = co.task(be.ops())
        for rep in range(2):
            _nan_outputs(crit)
            _nan_outputs(be)
            torch.cuda.synchronize()
            tk = {co.submit(bt, False), co.submit(ct, True), co.submit(bt, False)}
            co.drain(60000)
            recs = {r.ticket: r for r in co.poll()}
            assert set(recs) == tk and all(r.status == 0 for r in recs.values())
            torch.cuda.synchronize()
            for n in (crit, be):
                for l, r in zip(n.layers, ref[n.name]):
                    assert bits(l.t["y"]) == r, (policy, rep, n.name, l.name)
    finally:
        co.shutdown()
