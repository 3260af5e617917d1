"""The allocation-free LayerNorm backward (merak_layernorm_bwd_noalloc) against
the entry point it mirrors (merak_layernorm_bwd with a caller scratch buffer),
through the C ABI: two calls in a row, the second smaller, so that the second
reads nothing the first left in the library's scratch array.  Same kernels in
the same order, so the results must be bit-identical; the oracle's LayerNorm
backward checks the values themselves.  Also: a size beyond the array is
rejected before anything is enqueued."""
import numpy as np
import pytest

import oracle
from paper_2206_04959_amd import binding as B
from tests.gpu_util import need_gpu, rel_err

pytestmark = pytest.mark.gpu


def _case(torch, rows, h, seed, dtype):
    g = torch.Generator(device="cpu").manual_seed(seed)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    mk = lambda *s, std=1.0, mean=0.0: (torch.randn(*s, generator=g) * std + mean).to(dt).cuda()  # noqa: E731
    x, dout, dres = mk(rows, h, std=2.0), mk(rows, h), mk(rows, h)
    gamma, beta = mk(h, std=0.1, mean=1.0), mk(h, std=0.1)
    y = torch.empty_like(x)
    mean = torch.empty(rows, dtype=torch.float32, device="cuda")
    rstd = torch.empty(rows, dtype=torch.float32, device="cuda")
    B.layernorm_fwd(x, gamma, beta, y, mean, rstd)
    return dict(x=x, dout=dout, dres=dres, gamma=gamma, mean=mean, rstd=rstd)


def _run(torch, c, noalloc, accumulate=False, seed_out=None):
    rows, h = c["x"].shape
    dx = torch.empty_like(c["x"])
    dg = torch.full((h,), 0.5, dtype=torch.float32, device="cuda")
    db = torch.full((h,), -0.25, dtype=torch.float32, device="cuda")
    if noalloc:
        B.layernorm_bwd_noalloc(c["dout"], c["x"], c["mean"], c["rstd"], c["gamma"], c["dres"], dx, dg, db,
                                accumulate=accumulate)
    else:
        scratch = torch.empty(2 * B.reduce_scratch_elems(rows, h), dtype=torch.float32, device="cuda")
        B.layernorm_bwd(c["dout"], c["x"], c["mean"], c["rstd"], c["gamma"], c["dres"], dx, dg, db, scratch,
                        accumulate=accumulate)
    torch.cuda.synchronize()
    return dx, dg, db


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_noalloc_matches_layernorm_bwd_twice(dtype):
    torch = need_gpu()
    # second call smaller (fewer rows and columns) than the first
    for call, (rows, h, acc) in enumerate(((8192, 3072, False), (1000, 1024, True))):
        print(f"[noalloc] {dtype} call {call}: rows {rows} h {h} accumulate {acc}", flush=True)
        c = _case(torch, rows, h, 7 + call, dtype)
        want = _run(torch, c, noalloc=False, accumulate=acc)
        got = _run(torch, c, noalloc=True, accumulate=acc)
        for w, g_, name in zip(want, got, ("dx", "dgamma", "dbeta")):
            assert torch.equal(w, g_), (call, name)
        # the values themselves, against the oracle's LayerNorm backward
        x = c["x"].double().cpu().numpy()
        mu = x.mean(-1, keepdims=True)
        rs = 1.0 / np.sqrt(((x - mu) ** 2).mean(-1, keepdims=True) + 1e-5)
        dz, dgam, dbet = oracle.layer_norm_backward(c["dout"].double().cpu().numpy(), (x - mu) * rs, rs,
                                                    c["gamma"].double().cpu().numpy())
        tol = 2e-2 if dtype == "bf16" else 1e-4
        base_g, base_b = (0.5, -0.25) if acc else (0.0, 0.0)
        assert rel_err(got[0].double().cpu().numpy(), c["dres"].double().cpu().numpy() + dz) < tol
        assert rel_err(got[1].double().cpu().numpy(), base_g + dgam) < tol
        assert rel_err(got[2].double().cpu().numpy(), base_b + dbet) < tol


def test_noalloc_rejects_sizes_beyond_its_scratch():
    torch = need_gpu()
    cap = B.noalloc_scratch_elems()
    h = 8192
    rows = (cap // (2 * h) + 1) * 64  # one 64-row group more than fits
    assert 2 * B.reduce_scratch_elems(rows, h) > cap
    x = torch.zeros((rows, h), dtype=torch.bfloat16, device="cuda")
    stats = torch.zeros(rows, dtype=torch.float32, device="cuda")
    vec = torch.zeros(h, dtype=torch.float32, device="cuda")
    gam = torch.zeros(h, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.MerakError) as e:
        B.layernorm_bwd_noalloc(x, x, stats, stats, gam, x, x, vec, vec)
    assert e.value.status == -5  # MERAK_ERR_WORKSPACE
