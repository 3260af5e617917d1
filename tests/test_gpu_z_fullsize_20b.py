"""Full-size parity of the 20B-shaped workload in bf16 (4 blocks, hidden 6144,
48 heads / 6 local at head_dim 128, FFN 24576 / 3072 local, seq 2048,
micro-batch 4 in 4 sub-micro-batches, recompute on every block), in the
benchmark's launch configuration, at the stated 2e-2 max-relative bar.

Of all workloads this one sits closest to the bar: its worst tensor (an LN1
input-gradient partial) is dominated by bf16 storage rounding, not by kernel
error (a CPU replay of the oracle with bf16 rounding at the path's storage
points reaches the same level).  The file name makes pytest collect it after
the other GPU tests."""
import pytest

from tests.test_gpu_fullsize import check_full_size

pytestmark = pytest.mark.gpu


def test_full_size_20b_bf16_matches_oracle():
    check_full_size("gpt-20b-tp8", "bf16")
