"""GPU parity of the dense path (spconv_forward_dense, fp32 MFMA) against the
oracle, with the layer tolerance 1e-5 * sum|w*x| + 1e-6 per output (both paths
accumulate in fp32; only the order differs). Cases cover one to four waves per
workgroup, several channel tiles, partial channel tiles (K not a multiple of
32), odd C (the zero pad channel), several LDS chunks, one to eight 32-pixel
blocks per wave, 1x1 and 3x3 filters, pool, residual and zero-bordered
outputs. Every case prints its name and plan before touching the GPU.
"""
import numpy as np
import pytest

import oracle
from paper_2005_04091_amd import synth

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


def say(*a):
    print("[case]", *a, flush=True)


def check_close(gpu, ref, ab, what=""):
    gpu = np.asarray(gpu, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    err = np.abs(gpu - ref)
    bad = err > REL_TOL * ab + ABS_TOL
    assert not bad.any(), f"{what}: {int(bad.sum())} of {bad.size} outputs out of tolerance, max err {err.max():.3e}"


# N, C, K, H, W, R, density, pool, residual
CASES = [
    (1, 4, 8, 6, 7, 3, 0.5, False, False),
    (2, 5, 40, 9, 11, 3, 0.6, True, False),
    (1, 3, 33, 14, 14, 3, 1.0, False, True),
    (2, 7, 130, 5, 6, 1, 0.7, False, False),
    (1, 66, 16, 4, 30, 3, 0.4, True, True),
    (1, 2, 4, 2, 2, 3, 1.0, True, False),
    (1, 3, 16, 3, 224, 3, 0.5, False, False),
    (2, 17, 64, 30, 58, 3, 0.3, False, False),
    (4, 64, 64, 28, 28, 3, 0.5, True, False),
    (1, 130, 20, 7, 9, 3, 0.5, False, False),
    (3, 32, 96, 16, 16, 3, 0.2, False, True),
    (2, 9, 200, 12, 12, 3, 0.5, True, True),
]


def _layer(i):
    N, C, K, H, W, R, d, pool, _ = CASES[i]
    return synth.random_layer(8000 + i, N, C, K, H, W, R, R, 1, 1 if R == 3 else 0, d, True, pool, True, False)


def _dense_layer(sp, layer):
    N, C, H, W, K, R, S = layer.shape
    return sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, layer.pad, True, layer.pool, path="dense")


@pytest.mark.parametrize("i", range(len(CASES)))
def test_dense_against_oracle(sp, i):
    import torch
    layer = _layer(i)
    N, C, H, W, K, R, S = layer.shape
    L = _dense_layer(sp, layer)
    use_res = CASES[i][8]
    res = np.random.default_rng(200 + i).uniform(-1, 1, (N, K, H, W)).astype(np.float32) if use_res else None
    say("dense", CASES[i], L.plan(N))
    xp = L.pad_input(torch.from_numpy(layer.x).cuda())
    kw = {}
    if use_res:
        kw = dict(residual=torch.from_numpy(np.pad(res, ((0, 0), (0, 0), (1, 1), (1, 1)))).cuda(), residual_pad=1)
    out = L.forward_padded(xp, **kw)
    torch.cuda.synchronize()
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 1, layer.pad, True, layer.pool, residual=res)
    check_close(out.cpu().numpy(), ref, ab, f"dense {CASES[i]}")


@pytest.mark.parametrize("i", [0, 1, 7, 8])
def test_dense_out_pad_bitwise(sp, i):
    """A zero-bordered output holds the plain call's values bit for bit."""
    import torch
    layer = _layer(i)
    N, C, H, W, K, R, S = layer.shape
    L = _dense_layer(sp, layer)
    say("dense out_pad", CASES[i], L.plan(N))
    xp = L.pad_input(torch.from_numpy(layer.x).cuda())
    plain = L.forward_padded(xp)
    buf = torch.full((N, K, L.Ho + 2, L.Wo + 2), float("nan"), device="cuda")
    L.forward_padded(xp, out=buf, out_pad=1)
    torch.cuda.synchronize()
    ref = np.pad(plain.cpu().numpy(), ((0, 0), (0, 0), (1, 1), (1, 1)))
    assert np.array_equal(buf.cpu().numpy().view(np.uint32), ref.view(np.uint32))


def test_dense_full_size_narrow(sp):
    """The deep narrow layer at density 0.5 (32 x 256 x 14x14, Beta(2,5) row
    skew) in the plan the benchmark runs, whole output tensor against the
    oracle, and the dispatcher's choice for it."""
    import torch
    layer = synth.make_layer("narrow_d0.5")
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False, path="auto", N=N)
    assert L.path == "dense"
    say("dense narrow_d0.5 full size", L.plan(N))
    out = L.run(torch.from_numpy(layer.x).cuda())
    torch.cuda.synchronize()
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 1, 1, True, False)
    check_close(out.cpu().numpy(), ref, ab, "narrow_d0.5 dense")


def test_dense_and_sparse_agree(sp):
    """Both paths on one layer (ResNet-shaped, small batch): each within the
    layer tolerance of the oracle."""
    import torch
    layer = synth.random_layer(77, 2, 64, 64, 56, 56, 3, 3, 1, 1, 0.3, True, False, True, False)
    N, C, H, W, K, R, S = layer.shape
    x = torch.from_numpy(layer.x).cuda()
    outs = {}
    for path in ("sparse", "dense"):
        L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False, path=path)
        say("agree", path, L.plan(N))
        outs[path] = L.run(x)
    torch.cuda.synchronize()
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 1, 1, True, False)
    for path, o in outs.items():
        check_close(o.cpu().numpy(), ref, ab, path)
