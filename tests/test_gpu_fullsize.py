"""Parity at the full workload sizes, in the launch configuration the benchmark
times (two streams, the preset's sub-micro-batch count and recompute mask):
every output tensor against the fp64 oracle run on the same seeded inputs."""
import time

import pytest

from paper_2206_04959_amd import synth
from tests.gpu_util import StageRun, compare, oracle_results

pytestmark = pytest.mark.gpu

FULL = ["gpt-8.3b-tp4", "gpt-2.5b-tp2", "gpt-20b-tp8", "gpt-1.5b-stage"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_stage_matches_oracle(name):
    shape = synth.PRESETS[name]
    print(f"[full-size parity] {name}: {shape}", flush=True)
    t0 = time.time()
    got = StageRun(shape).run().results()
    print(f"  gpu done in {time.time() - t0:.1f} s; running the oracle", flush=True)
    t0 = time.time()
    ref = oracle_results(shape)
    print(f"  oracle done in {time.time() - t0:.1f} s", flush=True)
    errs, bad = compare(got, ref, shape)
    top = sorted(errs.items(), key=lambda kv: -kv[1])[:5]
    print("  worst: " + ", ".join(f"{k}={v:.3e}" for k, v in top), flush=True)
    assert not bad, bad
