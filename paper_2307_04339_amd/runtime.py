"""Python view of the coordinator (argument marshalling over the C ABI).

    with Coordinator(policy="elastic") as co:
        t = co.task([op1, op2, ...])
        ticket = co.submit(t, critical=True, release_ns=..., deadline_ns=0)
        records = co.poll()
"""
from __future__ import annotations

import ctypes

from . import _lib as L

POLICY = {"elastic": L.POLICY_ELASTIC, "sequential": L.POLICY_SEQUENTIAL,
          "multistream": L.POLICY_MULTISTREAM, "ib": L.POLICY_IB}


def default_config(**kw) -> L.Config:
    c = L.Config()
    c.policy = L.POLICY_ELASTIC
    c.backend = L.BACKEND_HIP
    c.n_be_streams = 1
    c.inflight_depth = 1
    c.top_frac = 0.2
    c.max_blk_frac = 0.1
    c.max_pt_frac = 0.1
    c.quantum_us = 50.0
    c.inflight_us = 0.0
    c.busy_policy = 0
    c.log_launches = 0
    c.profile_reps = 3
    c.fake_n_cu = 8
    c.fake_slots_per_cu = 2
    c.fake_tile_ns = 1000.0
    c.fake_launch_ns = 2000.0
    c.graphs = 1
    c.release_guard = 0
    c.warm_critical = 0
    c.graph_chunk = 0
    c.arm_lead_us = 0.0
    c.segments = 0
    c.event_us = 0.0
    c.be_cu_reserve = 0
    c.whole_when_clear = 0
    c.whole_margin = 0.0
    c.fake_fail_launch = 0
    c.crit_cu_exclusive = 0
    for k, v in kw.items():
        if k == "policy" and isinstance(v, str):
            v = POLICY[v]
        if k == "backend" and isinstance(v, str):
            v = {"hip": L.BACKEND_HIP, "fake": L.BACKEND_FAKE}[v]
        setattr(c, k, v)
    return c


class Task:
    def __init__(self, handle, ops):
        self.handle = handle
        self.ops = list(ops)  # keep the ops (and their tensors) alive


class Coordinator:
    def __init__(self, **cfg):
        self.lib = L.load()
        self.cfg = default_config(**cfg)
        L.check(self.lib.miriam_init(ctypes.byref(self.cfg)), "miriam_init")
        self._open = True
        self.tasks = []

    def task(self, ops) -> Task:
        arr = (ctypes.c_void_p * len(ops))(*[o.handle.value if hasattr(o, "handle") else o for o in ops])
        h = ctypes.c_void_p()
        L.check(self.lib.miriam_task_create(arr, len(ops), ctypes.byref(h)), "miriam_task_create")
        t = Task(h, ops)
        self.tasks.append(t)
        return t

    def submit(self, task: Task, critical: bool, release_ns: int = 0, deadline_ns: int = 0) -> int:
        tk = ctypes.c_uint64()
        L.check(self.lib.miriam_submit(task.handle, 1 if critical else 0, int(release_ns), int(deadline_ns),
                                       ctypes.byref(tk)), "miriam_submit")
        return tk.value

    def poll(self, max_out: int = 4096):
        buf = (L.Completion * max_out)()
        n = L.check(self.lib.miriam_poll(buf, max_out), "miriam_poll")
        return [buf[i] for i in range(n)]

    def drain(self, timeout_ms: int = 60000) -> None:
        L.check(self.lib.miriam_drain(timeout_ms), "miriam_drain")

    def stats(self) -> L.Stats:
        s = L.Stats()
        L.check(self.lib.miriam_stats_get(ctypes.byref(s)), "miriam_stats_get")
        return s

    def launch_log(self, max_out: int = 1 << 16):
        out = []
        buf = (L.LaunchRecord * max_out)()
        while True:
            n = L.check(self.lib.miriam_launch_log(buf, max_out), "miriam_launch_log")
            out.extend(L.LaunchRecord.from_buffer_copy(buf[i]) for i in range(n))
            if n < max_out:
                return out

    def now_ns(self) -> int:
        return int(self.lib.miriam_now_ns())

    def shutdown(self) -> None:
        if self._open:
            L.check(self.lib.miriam_shutdown(), "miriam_shutdown")
            self._open = False
            for t in self.tasks:
                self.lib.miriam_task_destroy(t.handle)
            self.tasks = []

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.shutdown()
