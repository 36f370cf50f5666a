"""GPU parity for every compiled kernel instance: each case of
``variant_cases.CASES`` (one seeded layer per instance of the stride-1 sparse
kernel and of the dense kernel) runs through the library, its plan is asserted
to be that instance, and the whole output tensor is compared with the oracle
element by element at |gpu - oracle| <= 1e-5 * A + 1e-6 (A = sum of |w * x|
of that output, its max over the window when pooled)."""
import numpy as np
import pytest

import oracle
import variant_cases as vc

pytestmark = pytest.mark.gpu

REL_TOL = 1e-5
ABS_TOL = 1e-6


@pytest.fixture(scope="module")
def sp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2005_04091_amd import spconv
    return spconv


def check_close(gpu, ref, ab, what):
    gpu = np.asarray(gpu, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    err = np.abs(gpu - ref)
    tol = REL_TOL * ab + ABS_TOL
    bad = err > tol
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outputs out of tolerance; worst at {i}: "
                             f"gpu={gpu[i]!r} oracle={ref[i]!r} A={ab[i]!r}")


@pytest.mark.parametrize("case", vc.CASES, ids=[f"{c[0]}{c[1]}" for c in vc.CASES])
def test_instance_against_oracle(sp, case):
    """Each instance against the oracle; stride-1 instances in both forms (the
    plain CSR walk and the lowered entry stream, for "s1t" cases in its form
    with several work items per workgroup), which must agree bit for bit
    (same entries, same summation order)."""
    import torch
    kind, variant, N, C, K, H, W, d, skew, pool, seed = case
    layer = vc.case_layer(case)
    R, S = layer.w.shape[2], layer.w.shape[3]
    print("[case]", kind, variant, (N, C, K, H, W, R, S), "density", d, "skew", skew, flush=True)
    outs = {}
    ref = ab = None
    for lowered in ((False, True) if kind != "dense" else (False,)):
        L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, layer.pad, True, pool,
                               path="dense" if kind == "dense" else "sparse", lowered=lowered)
        plan = L.plan(N)
        got = (R, S, plan["pixels_per_lane"], int(pool)) if kind == "dense" else \
            (plan["pixels_per_lane"], plan["images_per_group"], plan["channels_per_wave"], int(pool))
        assert got == variant, (got, plan)
        assert (L.lowered(N) is not None) == lowered
        if kind != "dense":  # the lowered "s1t" cases run several work items per workgroup
            assert (plan["launch_workgroups"] < plan["workgroups"]) == (lowered and kind == "s1t"), plan
        print("[case]   lowered" if lowered else "[case]   plain", flush=True)
        out = L.run(torch.from_numpy(layer.x).cuda())
        torch.cuda.synchronize()
        outs[lowered] = out.cpu().numpy()
        if ref is None:
            ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 1, layer.pad, True, pool)
        check_close(outs[lowered], ref, ab, f"{kind} {variant} lowered={lowered}")
    if len(outs) == 2:
        assert np.array_equal(outs[False].view(np.uint32), outs[True].view(np.uint32))
