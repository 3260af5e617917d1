"""Whole-stage parity of the HIP path against the fp64 oracle, through the C ABI,
plus the schedule properties the method guarantees (split independence,
recomputation equality, determinism) and call-order errors."""
import numpy as np
import pytest

from paper_2206_04959_amd import binding as B
from paper_2206_04959_amd import synth
from tests.gpu_util import ELEM_TOL_FP32, StageRun, compare, elem_err, need_gpu, oracle_results

pytestmark = pytest.mark.gpu

# Small shapes that still span several GEMM tiles, attention tiles and a ragged
# 128-tile edge (3h/t = 384, h = 320 ...), each head_dim, tensor parallel shards.
SMALL = {
    "tiny-fp32": synth.TINY,
    "tiny-bf16": synth.TINY.replace(dtype="bf16"),
    "tiny-fp32-n2-rc": synth.TINY.replace(n_sub=2, recompute_mask=1),
    "d64-t2-bf16": synth.StageShape("d64", n_blocks=3, hidden=512, n_heads=8, ffn=2048, seq_len=256,
                                    micro_batch=4, tp_degree=2, n_sub=2, recompute_mask=0b010, seed=31),
    "d96-bf16": synth.StageShape("d96", n_blocks=2, hidden=384, n_heads=4, ffn=1536, seq_len=192,
                                 micro_batch=2, tp_degree=1, n_sub=2, recompute_mask=0b01, seed=32),
    "d96-fp32": synth.StageShape("d96f", n_blocks=2, hidden=384, n_heads=4, ffn=1536, seq_len=128,
                                 micro_batch=2, tp_degree=1, n_sub=2, recompute_mask=0b10, dtype="fp32",
                                 x_std=1.0, seed=33),
    "d128-t4-bf16": synth.StageShape("d128", n_blocks=2, hidden=1024, n_heads=8, ffn=4096, seq_len=128,
                                     micro_batch=4, tp_degree=4, n_sub=4, recompute_mask=0b11, seed=34),
    # three sub-micro-batches: the two streams carry two and one of them, so
    # the per-stream grouped launches have unequal member counts
    "d64-n3-bf16": synth.StageShape("d64n3", n_blocks=2, hidden=256, n_heads=4, ffn=1024, seq_len=128,
                                    micro_batch=6, tp_degree=1, n_sub=3, recompute_mask=0b10, seed=35),
    # the smallest stage the boundary accepts: one block, one head of 64, one
    # 64-token sequence (every GEMM a single partial tile, one attention block,
    # one reduction segment)
    "min-bf16": synth.StageShape("min", n_blocks=1, hidden=64, n_heads=1, ffn=64, seq_len=64, micro_batch=1,
                                 tp_degree=1, n_sub=1, recompute_mask=0b1, seed=36),
    "min-fp32": synth.StageShape("minf", n_blocks=1, hidden=64, n_heads=1, ffn=64, seq_len=64, micro_batch=1,
                                 tp_degree=1, n_sub=1, recompute_mask=0b0, dtype="fp32", seed=37),
    # the largest block count (64), every other block recomputed, bit 63 included
    "max-blocks-fp32": synth.StageShape("maxl", n_blocks=64, hidden=64, n_heads=1, ffn=64, seq_len=64,
                                        micro_batch=2, tp_degree=1, n_sub=2, recompute_mask=0xAAAAAAAAAAAAAAAA,
                                        dtype="fp32", seed=38),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_stage_matches_oracle(name):
    shape = SMALL[name]
    print(f"[stage parity] {name}: {shape}", flush=True)
    got = StageRun(shape).run().results()
    ref = oracle_results(shape)
    errs, bad = compare(got, ref, shape)
    worst = max(errs, key=errs.get)
    print(f"  worst {worst} = {errs[worst]:.3e}", flush=True)
    assert not bad, bad
    # elementwise relative error with a 1e-3 max|o| floor: gates the tiny fp32 workload
    eerrs, ebad = compare(got, ref, shape, tol=ELEM_TOL_FP32, metric=elem_err)
    eworst = max(eerrs, key=eerrs.get)
    print(f"  elementwise (floor 1e-3 max): worst {eworst} = {eerrs[eworst]:.3e}", flush=True)
    if name == "tiny-fp32":
        assert not ebad, ebad


def test_recompute_gives_bit_identical_gradients():
    base = SMALL["d64-t2-bf16"]
    a = StageRun(base.replace(recompute_mask=0)).run().raw()
    b = StageRun(base.replace(recompute_mask=0b111)).run().raw()
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_recompute_on_its_own_streams_overlapping_the_backward():
    """Recomputation issued on other streams than the backward (the backward
    of each recomputed block waits for that block only) gives the same bits."""
    base = SMALL["d64-t2-bf16"].replace(recompute_mask=0b011)
    a = StageRun(base).run().raw()
    b = StageRun(base, rc_streams=True).run().raw()
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def test_sub_micro_batch_split_and_streams_do_not_change_results():
    base = SMALL["d64-t2-bf16"]
    ref = StageRun(base.replace(n_sub=1), streams=1).run().raw()
    for n, streams in ((2, 2), (4, 2), (4, 1)):
        got = StageRun(base.replace(n_sub=n), streams=streams).run().raw()
        for k in ref:
            assert np.array_equal(ref[k], got[k]), (n, streams, k)


def test_grouped_launches_do_not_change_results():
    """Sub-micro-batch counts whose per-stream groups hold 1, 2 or 3 members
    (grouped GEMM and attention launches) give the unsplit bits."""
    base = SMALL["d64-n3-bf16"]
    ref = StageRun(base.replace(n_sub=1), streams=1).run().raw()
    for n in (2, 3, 6):
        got = StageRun(base.replace(n_sub=n)).run().raw()
        for k in ref:
            assert np.array_equal(ref[k], got[k]), (n, k)


def test_runs_are_deterministic_and_accumulate_adds():
    torch = need_gpu()
    shape = SMALL["d96-bf16"]
    r = StageRun(shape)
    a = r.run().raw()
    b = r.run().raw()
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    g1 = r.grads.clone()
    r.run(accumulate=True)
    assert torch.equal(r.grads, g1 + g1) or torch.allclose(r.grads, 2 * g1, rtol=1e-6, atol=0)


def test_without_hand_off_buffers():
    shape = SMALL["d96-bf16"]
    ref = StageRun(shape).run().raw()
    got = StageRun(shape, with_partials=False).run().raw()
    for k in ("y", "dx", "grads"):
        assert np.array_equal(ref[k], got[k]), k


def test_call_order_errors():
    torch = need_gpu()
    shape = SMALL["tiny-fp32-n2-rc"]
    r = StageRun(shape)
    st = r.stage
    with pytest.raises(B.MerakError) as e:
        st.bwd(r.params, r.dy, r.dx, r.grads)
    assert e.value.status == -3
    with pytest.raises(B.MerakError) as e:
        st.recompute(r.params)
    assert e.value.status == -3
    st.fwd(r.params, r.x, r.y)
    with pytest.raises(B.MerakError) as e:  # recompute pending
        st.bwd(r.params, r.dy, r.dx, r.grads)
    assert e.value.status == -3
    st.recompute(r.params)
    # a second handle sharing the recompute area takes it over
    other = B.Stage(shape, recompute_area=st.recompute_area)
    other.fwd(r.params, r.x, r.y)
    other.recompute(r.params)
    with pytest.raises(B.MerakError) as e:
        st.bwd(r.params, r.dy, r.dx, r.grads)
    assert e.value.status == -3
    other.bwd(r.params, r.dy, r.dx, r.grads)
    st.recompute(r.params)
    st.bwd(r.params, r.dy, r.dx, r.grads)
    torch.cuda.synchronize()
    with pytest.raises(B.MerakError) as e:  # consumed
        st.bwd(r.params, r.dy, r.dx, r.grads)
    assert e.value.status == -3
    other.close()


def test_failed_launch_leaves_handle_refusing_dependent_calls():
    """An injected launch failure (merak_debug_fail_after: the call returns
    MERAK_ERR_HIP instead of making the launch) part-way through fwd, recompute
    or bwd leaves the handle refusing the calls that would read what the failed
    call did not finish; after clearing the injection the handle works and
    gives the same bits as a handle that never failed."""
    torch = need_gpu()
    shape = SMALL["d64-t2-bf16"].replace(recompute_mask=0b011)
    ref = StageRun(shape).run().raw()
    r = StageRun(shape)
    st = r.stage
    try:
        B.debug_fail_after(3)
        with pytest.raises(B.MerakError) as e:
            st.fwd(r.params, r.x, r.y)
        assert e.value.status == -6
        B.debug_fail_after(-1)
        for call in (lambda: st.recompute(r.params), lambda: st.bwd(r.params, r.dy, r.dx, r.grads)):
            with pytest.raises(B.MerakError) as e:
                call()
            assert e.value.status == -3
        st.fwd(r.params, r.x, r.y)
        B.debug_fail_after(2)
        with pytest.raises(B.MerakError) as e:
            st.recompute(r.params)
        assert e.value.status == -6
        B.debug_fail_after(-1)
        with pytest.raises(B.MerakError) as e:  # recomputation incomplete
            st.bwd(r.params, r.dy, r.dx, r.grads)
        assert e.value.status == -3
        st.recompute(r.params)
        B.debug_fail_after(5)
        with pytest.raises(B.MerakError) as e:
            st.bwd(r.params, r.dy, r.dx, r.grads)
        assert e.value.status == -6
        B.debug_fail_after(-1)
        with pytest.raises(B.MerakError) as e:  # consumed by the failed call
            st.bwd(r.params, r.dy, r.dx, r.grads)
        assert e.value.status == -3
    finally:
        B.debug_fail_after(-1)
    torch.cuda.synchronize()
    got = r.run().raw()
    for k in ref:
        assert np.array_equal(ref[k], got[k]), k


@pytest.mark.parametrize("name", ["tiny-bf16", "tiny-fp32"])
def test_nonfinite_scan_of_stage_outputs(name):
    """Failure detection: a clean step leaves no NaN/Inf in y, dx or the
    gradients; one NaN planted in the stage input (from the host) shows in the
    scan of y, dx and the gradients."""
    shape = SMALL[name]
    print(f"[nonfinite scan] {name}", flush=True)
    run = StageRun(shape)
    torch = run.torch
    count = torch.zeros(1, dtype=torch.int64, device="cuda")

    def scan(t):
        B.count_nonfinite(t, count)
        torch.cuda.synchronize()
        return int(count.item())

    run.run()
    assert scan(run.y) == 0 and scan(run.dx) == 0 and scan(run.grads) == 0
    x = run.x.view(-1)
    x[x.numel() // 3] = float("nan")  # one token's hidden state
    torch.cuda.synchronize()
    run.run()
    ny, ndx, ng = scan(run.y), scan(run.dx), scan(run.grads)
    print(f"  non-finite after one NaN in x: y {ny}, dx {ndx}, grads {ng}", flush=True)
    assert ny >= shape.hidden and ndx > 0 and ng > 0
