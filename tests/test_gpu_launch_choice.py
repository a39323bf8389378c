"""How planned transfers pick their launch (kvx_set_launch_choice), on the
GPU through the product library.  In the measured mode the first six calls
of a key take the sweep and the persistent grid in turn, the next four
(timed) the sweep, the grid, the grid and the sweep, and once their timings
are in, every later call takes one launch, the same each time; a new key,
or setting the mode again, starts over; other records on the same pools
share the pools' measurement.  The fixed modes always take their
launch, a call captured in a HIP graph records no events and takes the
sweep, two host threads can measure one key at once, and every call's
result is the oracle's, bit for bit."""
import numpy as np
import pytest

import cases
from paper_2606_31093_amd.kvx import LAUNCH_GRID, LAUNCH_SWEEP
from runner import initial_bytes, run_oracle

pytestmark = pytest.mark.gpu

# launches of the first calls of a key in the measured mode (kvx.h): six
# untimed, then four timed
MEASURE = [LAUNCH_SWEEP, LAUNCH_GRID] * 3 + [LAUNCH_SWEEP, LAUNCH_GRID, LAUNCH_GRID, LAUNCH_SWEEP]


@pytest.fixture
def kvx():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31093_amd import kvx
    kvx.lib()
    kvx.kvx_set_launch_choice(kvx.CHOOSE_MEASURED)
    yield kvx
    kvx.kvx_set_launch_choice(kvx.CHOOSE_MEASURED)


class Case:
    """A transfer the product library can sweep (256 KiB pages), its pools on
    the GPU and the oracle's result."""

    def __init__(self, kvx, seed, ld="PLCTHD"):
        import torch
        spec = [(0, 0, 200, None), (5, 70, 333, None), (63, 1, 1, None), (10, 64, 128, 0)]
        wl = cases.transfer_case("LPCTHD", ld, 64, 64, seed=seed, e=2, D=128, L=3, C=2, H=8, spec=spec)
        self.kvx, self.st = kvx, wl.steps[0]
        self.S, self.D = wl.sides["A"], wl.sides["B"]
        init = initial_bytes(wl)
        self.want = run_oracle(wl, init)[0]["B"]
        self.a = torch.from_numpy(init["A"]).cuda()
        self.b = torch.from_numpy(init["B"]).cuda()
        self.b0 = self.b.clone()
        self.spt, self.dpt = kvx.device_table(self.st.src_pt), kvx.device_table(self.st.dst_pt)
        self.reqs = kvx.device_reqs(self.st.reqs)
        self.plan, self.pages, self.tokens = kvx.device_plan(self.st.reqs, self.S.T, self.D.T)
        self.err = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.wl, self.init = wl, init
        self.subset = None

    def use_records(self, rows):
        """Later calls move only these records (rows of the case's own),
        over the same pools and tables."""
        import dataclasses
        if rows is None:
            self.subset = None
            return
        st = dataclasses.replace(self.st, reqs=np.asarray(rows, np.int64).reshape(-1, 6))
        wl = dataclasses.replace(self.wl, steps=[st])
        plan, pages, tokens = self.kvx.device_plan(st.reqs, self.S.T, self.D.T)
        self.subset = (self.kvx.device_reqs(st.reqs), plan, pages, tokens, run_oracle(wl, self.init)[0]["B"])

    def call(self, check=True):
        """One planned call into a fresh copy of the destination; returns the
        launch it took."""
        import torch
        reqs, plan, pages, tokens, want = self.subset or (self.reqs, self.plan, self.pages, self.tokens,
                                                          self.want)
        self.b.copy_(self.b0)
        self.err.zero_()
        self.kvx.kvx_transfer_planned(self.a, self.S, self.b, self.D, self.spt, self.dpt, reqs, plan, pages,
                                      tokens, None, self.err)
        launch = self.kvx.kvx_last_launch()
        if check:
            torch.cuda.synchronize()
            assert int(self.err.item()) == 0
            assert np.array_equal(self.b.cpu().numpy(), want)
        return launch


def test_measured_sequence(kvx):
    import torch
    c = Case(kvx, seed=41)
    S, G = kvx.LAUNCH_SWEEP, kvx.LAUNCH_GRID
    assert [c.call() for _ in range(10)] == MEASURE
    torch.cuda.synchronize()
    decided = c.call()
    assert decided in (S, G)
    assert [c.call() for _ in range(4)] == [decided] * 4


def test_calls_sweep_until_the_timings_are_in(kvx):
    """With the stream held busy (a bounded spin of about 50 ms queued first),
    the calls after the two timed ones find the timings still pending and
    sweep; after a synchronize the decision comes at the next call."""
    import torch
    c = Case(kvx, seed=43)
    S, G = kvx.LAUNCH_SWEEP, kvx.LAUNCH_GRID
    torch.cuda._sleep(100_000_000)
    launches = [c.call(check=False) for _ in range(12)]
    assert launches == MEASURE + [S, S]
    torch.cuda.synchronize()
    decided = c.call()
    assert decided in (S, G)
    assert c.call() == decided


def test_keys_are_separate_and_setting_the_mode_starts_over(kvx):
    import torch
    S, G = kvx.LAUNCH_SWEEP, kvx.LAUNCH_GRID
    c1, c2 = Case(kvx, seed=45), Case(kvx, seed=47, ld="PLCHTD")
    assert [c1.call() for _ in range(10)] == MEASURE
    assert [c2.call() for _ in range(10)] == MEASURE         # another key: its own sequence
    torch.cuda.synchronize()
    assert c1.call() in (S, G)
    kvx.kvx_set_launch_choice(kvx.CHOOSE_MEASURED)           # forgets every key
    assert [c1.call() for _ in range(10)] == MEASURE


def test_other_records_on_the_same_pools_share_the_measurement(kvx):
    """A serving loop moves other requests in every call: calls on the same
    pools count toward one measurement whatever their records, and keep its
    decision."""
    import torch
    c = Case(kvx, seed=61)
    S, G = kvx.LAUNCH_SWEEP, kvx.LAUNCH_GRID
    rows = c.st.reqs.tolist()
    launches = []
    for i in range(10):
        c.use_records(rows[: 1 + i % 3] if i % 2 else None)   # the full set, or its first 1-3 records
        launches.append(c.call())
    assert launches == MEASURE
    torch.cuda.synchronize()
    c.use_records(rows[:2])
    decided = c.call()
    assert decided in (S, G)
    c.use_records(None)
    assert [c.call() for _ in range(3)] == [decided] * 3


@pytest.mark.parametrize("mode,launch", [("CHOOSE_SWEEP", "LAUNCH_SWEEP"), ("CHOOSE_GRID", "LAUNCH_GRID")])
def test_fixed_modes(kvx, mode, launch):
    kvx.kvx_set_launch_choice(getattr(kvx, mode))
    c = Case(kvx, seed=49)
    assert [c.call() for _ in range(5)] == [getattr(kvx, launch)] * 5


def test_unplanned_and_small_calls_take_the_grid(kvx):
    """Without a plan, or below the sweep's page size, there is nothing to
    choose: the persistent grid, whatever the mode."""
    import torch
    c = Case(kvx, seed=51)
    for _ in range(4):
        c.b.copy_(c.b0)
        kvx.kvx_transfer(c.a, c.S, c.b, c.D, c.spt, c.dpt, c.reqs, c.err)
        assert kvx.kvx_last_launch() == kvx.LAUNCH_GRID
    torch.cuda.synchronize()
    assert np.array_equal(c.b.cpu().numpy(), c.want)
    small = cases.transfer_case("LPCTHD", "LPCTHD", 16, 16, seed=53)
    st = small.steps[0]
    S, D = small.sides["A"], small.sides["B"]
    init = initial_bytes(small)
    a, b = torch.from_numpy(init["A"]).cuda(), torch.from_numpy(init["B"]).cuda()
    plan, pages, tokens = kvx.device_plan(st.reqs, S.T, D.T)
    for _ in range(4):
        kvx.kvx_transfer_planned(a, S, b, D, kvx.device_table(st.src_pt), kvx.device_table(st.dst_pt),
                                 kvx.device_reqs(st.reqs), plan, pages, tokens, None, c.err)
        assert kvx.kvx_last_launch() == kvx.LAUNCH_GRID
    torch.cuda.synchronize()
    assert np.array_equal(b.cpu().numpy(), run_oracle(small, init)[0]["B"])


def test_captured_call_records_nothing_and_replays_exact(kvx):
    """Captured in a HIP graph (no events may be recorded there), a call of a
    key still in measurement takes the sweep; the replays are exact, and the
    key's measurement goes on outside the capture."""
    import torch
    c = Case(kvx, seed=55)
    S, G = kvx.LAUNCH_SWEEP, kvx.LAUNCH_GRID
    assert c.call() == S                                     # first call of the key
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        kvx.kvx_transfer_planned(c.a, c.S, c.b, c.D, c.spt, c.dpt, c.reqs, c.plan, c.pages, c.tokens,
                                 None, c.err)
        captured = kvx.kvx_last_launch()
    assert captured == S
    for _ in range(3):
        c.b.copy_(c.b0)
        c.err.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(c.err.item()) == 0
        assert np.array_equal(c.b.cpu().numpy(), c.want)
    assert [c.call() for _ in range(9)] == MEASURE[1:]       # the measurement goes on
    torch.cuda.synchronize()
    assert c.call() in (S, G)


def test_two_threads_measure_one_key(kvx):
    """Two host threads on two streams make the calls of one key while it is
    measured (both write the same bytes into the same pools).  Every call
    returns, the result is the oracle's, and afterwards the key keeps one
    launch."""
    import threading

    import torch
    c = Case(kvx, seed=57)
    S, G = kvx.LAUNCH_SWEEP, kvx.LAUNCH_GRID
    c.b.copy_(c.b0)
    torch.cuda.synchronize()
    failures = []

    def worker():
        s = torch.cuda.Stream()
        try:
            with torch.cuda.stream(s):
                for _ in range(12):
                    kvx.kvx_transfer_planned(c.a, c.S, c.b, c.D, c.spt, c.dpt, c.reqs, c.plan, c.pages,
                                             c.tokens, None, c.err, stream=s)
            s.synchronize()
        except Exception as e:           # reported below, on the test's thread
            failures.append(e)

    threads = [threading.Thread(target=worker) for _ in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not failures, failures
    assert int(c.err.item()) == 0
    assert np.array_equal(c.b.cpu().numpy(), c.want)
    decided = c.call()
    assert decided in (S, G)
    assert [c.call() for _ in range(3)] == [decided] * 3
