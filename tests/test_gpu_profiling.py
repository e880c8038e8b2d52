"""Per-phase event timing: the factors do not depend on whether or how launches are timed;
mode 1 times every phase, mode 2 only the launches that build the normal equations (the
gather kernels, and above D = 20 the fused row kernel); other modes are refused."""
import numpy as np
import pytest

import workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")


@pytest.mark.parametrize("D", [20, 48])
def test_profiling_modes(D):
    from paper_1108_2580_amd import ALS, ALSError, lib

    M, N = 3000, 2000
    rng = np.random.default_rng(31 + D)
    deg = rng.integers(0, 120, size=M)
    ptr, col, val = workload.make_custom(M, N, deg, seed=41 + D)
    U0, V0 = workload.init_factors(M, N, D, seed=43 + D)
    print(f"profiling modes: {M} x {N}, nnz {int(ptr[-1])}, D {D}", flush=True)
    res, prof = {}, {}
    # rows above 64 ratings split into chunks of 32, so that the gather phase has launches
    # above D = 20 too
    with ALS(M, N, ptr, col, val, D, tuning=dict(hub_threshold=64, chunk=32)) as als:
        assert als.plan_stats("users")["split_rows"] > 0
        for mode in (0, 1, 2):
            if mode:
                als.set_profiling(True, gram_only=(mode == 2))
            u, v = dev(U0), dev(V0)
            als.half_sweep("items", u, 0.065, v, allow_flagged=True)
            als.half_sweep("users", v, 0.065, u, allow_flagged=True)
            if mode:
                prof[mode] = als.profile()
                als.set_profiling(False)
            res[mode] = (u.cpu().numpy(), v.cpu().numpy())
        with pytest.raises(ALSError):
            als._check(lib.als_set_profiling(als._h, 3))
    for mode in (1, 2):
        for a, b in zip(res[0], res[mode]):
            assert np.array_equal(a, b)
    p1, p2 = prof[1], prof[2]
    print(f"  mode 1 {p1}\n  mode 2 {p2}", flush=True)
    assert p1["stage"][1] == 2 and p1["reduce"][1] == 2
    assert p1["gather"][1] >= 2 and p1["solve"][1] >= 2
    assert p2["stage"][1] == 0 and p2["reduce"][1] == 0 and p2["residual"][1] == 0
    assert p2["gather"][1] == p1["gather"][1]
    assert p2["solve"][1] == (0 if D <= 20 else p1["solve"][1])
