"""Pipeline schedules of Sec. 5.1: the oracle pinned against the paper's bubble
ratios and structural properties, and the C implementation against the oracle."""
import pytest

from oracle import schedule as S
from paper_2206_04959_amd import binding as B

KINDS = {"1f1b": B.SCHED_1F1B, "early": B.SCHED_EARLY_RECOMPUTE, "scp": B.SCHED_SCP}
TYPE = {"F": B.OP_FWD, "R": B.OP_RECOMPUTE, "B": B.OP_BWD, "RB": B.OP_RECOMPUTE_BWD}
RATIO = {
    "1f1b": lambda s, m: (s - 1) / m,              # 4(s-1) T_m of bubble over 4 m T_m
    "early": lambda s, m: 3 * (s - 1) / (4 * m),   # recomputation moved ahead of the gradient
    "scp": lambda s, m: 3 * (s - 2) / (4 * m),     # critical path shifted to the penultimate stage
}


# --- pins of the oracle ----------------------------------------------------

@pytest.mark.parametrize("kind", sorted(KINDS))
def test_bubble_ratios_match_the_paper(kind):
    for s in range(2, 17):
        for m in range(s, 3 * s + 1):
            if kind == "scp" and s == m == 2:
                continue  # two micro-batches cannot fill the tail (makespan 9 T_m, not 8)
            assert S.bubble_ratio(kind, s, m) == pytest.approx(RATIO[kind](s, m), abs=1e-12), (s, m)


def test_scp_tail_exception_is_a_true_lower_bound():
    # s = m = 2: the last stage's second backward ends at 7 T_m at the earliest
    # (F0 1-2, B0 2-4, F1 4-5, B1 5-7), and stage 0 still needs 2 T_m for B1.
    assert S.simulate("scp", 2, 2)[0] == 9.0


@pytest.mark.parametrize("kind", sorted(KINDS))
@pytest.mark.parametrize("s,m", [(1, 3), (2, 5), (4, 4), (4, 9), (8, 16), (5, 3)])
def test_every_dependency_respected_and_every_op_once(kind, s, m):
    makespan, busy, fin = S.simulate(kind, s, m)
    for i in range(s):
        ops = S.stage_ops(kind, s, m, i)
        assert sorted(j for op, j in ops if op == "F") == list(range(m))
        assert sorted(j for op, j in ops if op in ("B", "RB")) == list(range(m))
        rc = sorted(j for op, j in ops if op == "R")
        assert rc == ([] if kind == "1f1b" or (kind == "scp" and i == s - 1) else list(range(m)))
        for j in range(m):
            start_f = fin[("F", i, j)] - S.COST["F"]
            if i > 0:
                assert start_f >= fin[("F", i - 1, j)] - 1e-12
            bcost = S.COST["RB"] if kind == "1f1b" else S.COST["B"]
            start_b = fin[("B", i, j)] - bcost
            if i < s - 1:
                assert start_b >= fin[("B", i + 1, j)] - 1e-12
            assert start_b >= fin[("F", i, j)] - 1e-12
            if ("R", i, j) in fin:
                assert start_b >= fin[("R", i, j)] - 1e-12
    assert max(busy) <= makespan


def test_in_flight_micro_batches():
    # stage i of 1F1B holds at most s - i micro-batches; SCP's penultimate stage
    # holds one more (the forward brought ahead), its last stage exactly one.
    for kind in KINDS:
        s, m = 6, 12
        for i in range(s):
            live, peak = 0, 0
            for op, j in S.stage_ops(kind, s, m, i):
                if op == "F":
                    live += 1
                    peak = max(peak, live)
                elif op in ("B", "RB"):
                    live -= 1
            extra = 1 if (kind == "scp" and i == s - 2) else 0
            assert peak == min(s - i, m) + extra, (kind, i)


def test_scp_penultimate_order():
    assert S.stage_ops("scp", 4, 5, 2)[:5] == [("F", 0), ("F", 1), ("R", 0), ("F", 2), ("B", 0)]
    assert S.stage_ops("scp", 4, 5, 3)[:4] == [("F", 0), ("B", 0), ("F", 1), ("B", 1)]


# --- the C implementation against the oracle ------------------------------

@pytest.mark.parametrize("kind", sorted(KINDS))
@pytest.mark.parametrize("s", [1, 2, 3, 4, 7, 8, 16])
def test_abi_op_lists_match_oracle(kind, s):
    for m in range(1, 3 * s + 2):
        for i in range(s):
            ref = [(TYPE[op], j) for op, j in S.stage_ops(kind, s, m, i)]
            assert B.schedule_stage(KINDS[kind], s, m, i) == ref, (s, m, i)


@pytest.mark.parametrize("kind", sorted(KINDS))
@pytest.mark.parametrize("s,m", [(1, 1), (2, 2), (4, 5), (4, 8), (8, 16), (16, 40), (5, 3)])
def test_abi_simulation_matches_oracle(kind, s, m):
    mk, busy = B.schedule_simulate(KINDS[kind], s, m)
    ref_mk, ref_busy, _ = S.simulate(kind, s, m)
    assert mk == ref_mk and busy == ref_busy
    # other costs (a forward of 1, recompute 0.8, backward 2.3)
    cost = {"F": 1.0, "R": 0.8, "B": 2.3, "RB": 3.1}
    mk, busy = B.schedule_simulate(KINDS[kind], s, m, 1.0, 0.8, 2.3)
    ref_mk, ref_busy, _ = S.simulate(kind, s, m, cost)
    assert mk == pytest.approx(ref_mk, abs=1e-9) and busy == pytest.approx(ref_busy, abs=1e-9)


def test_abi_schedule_errors():
    import ctypes
    L = B.lib()
    n = ctypes.c_int()
    buf = (ctypes.c_int32 * 4)()
    assert L.merak_schedule_stage(7, 4, 4, 0, buf, 4, ctypes.byref(n)) == -1
    assert L.merak_schedule_stage(0, 0, 4, 0, buf, 4, ctypes.byref(n)) == -2
    assert L.merak_schedule_stage(0, 4, 4, 4, buf, 4, ctypes.byref(n)) == -1
    assert L.merak_schedule_stage(0, 4, 4, 0, buf, 4, ctypes.byref(n)) == -5 and n.value == 8


@pytest.mark.parametrize("kind", sorted(KINDS))
def test_abi_inflight_matches_oracle(kind):
    """The handles merak_schedule_run needs: the peak of micro-batches between
    their forward and their backward in the oracle's op list."""
    for s in (1, 2, 3, 4, 8):
        for m in range(1, 3 * s + 2):
            for i in range(s):
                live, peak = 0, 0
                for op, j in S.stage_ops(kind, s, m, i):
                    if op == "F":
                        live += 1
                        peak = max(peak, live)
                    elif op in ("B", "RB"):
                        live -= 1
                assert B.schedule_inflight(KINDS[kind], s, m, i) == peak, (s, m, i)
