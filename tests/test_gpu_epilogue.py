"""GPU tests of the epilogue options (spconv_forward_ex): a zero border around
the stored planes (the next layer's padded input, so chained layers skip the
padding pass) and a residual added before the activation (the shortcut of a
ResNet basic block).

The padded output must hold exactly the values of the plain call (same kernel,
same arithmetic) inside a border of +0.0; the residual is checked against the
oracle, whose sum of |w*x| includes |residual|. Every case prints its name and
shape before touching the GPU.
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
    tol = REL_TOL * ab + ABS_TOL
    bad = err > tol
    assert not bad.any(), f"{what}: {int(bad.sum())} of {bad.size} outputs out of tolerance, max err {err.max():.3e}"


# N, C, K, H, W, stride, pad, density, pool  (stride-1 tilings of one and several
# tiles and images per group, and the any-stride kernel)
CASES = [
    (1, 16, 16, 16, 16, 1, 1, 0.2, False),
    (2, 8, 16, 61, 70, 1, 1, 0.2, True),
    (3, 12, 10, 19, 23, 1, 1, 0.3, False),
    (16, 3, 130, 2, 2, 1, 1, 0.3, True),
    (8, 3, 520, 2, 2, 1, 1, 0.3, False),
    (2, 5, 7, 9, 8, 2, 1, 0.4, False),
    (2, 5, 3, 10, 12, 2, 1, 0.4, True),
    (1, 4, 4, 5, 300, 1, 1, 0.3, False),
]


def _layer(i, case):
    N, C, K, H, W, stride, pad, d, pool = case
    return synth.random_layer(7000 + i, N, C, K, H, W, 3, 3, stride, pad, d, True, pool, True, False)


@pytest.mark.parametrize("out_pad", [1, 2])
@pytest.mark.parametrize("i", range(len(CASES)))
def test_out_pad_matches_plain_call_bitwise(sp, i, out_pad):
    import torch
    layer = _layer(i, CASES[i])
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, layer.stride, layer.pad, layer.relu, layer.pool)
    say("out_pad", out_pad, CASES[i], L.plan(N))
    xp = L.pad_input(torch.from_numpy(layer.x).cuda())
    plain = L.forward_padded(xp)
    Hs, Ws = L.Ho, L.Wo
    buf = torch.full((N, K, Hs + 2 * out_pad, Ws + 2 * out_pad), float("nan"), device="cuda")
    L.forward_padded(xp, out=buf, out_pad=out_pad)
    torch.cuda.synchronize()
    got = buf.cpu().numpy()
    ref = np.pad(plain.cpu().numpy(), ((0, 0), (0, 0), (out_pad, out_pad), (out_pad, out_pad)))
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), "padded output differs from pad(plain output)"


@pytest.mark.parametrize("res_pad", [0, 1, 2])
@pytest.mark.parametrize("i", range(len(CASES)))
def test_residual_against_oracle(sp, i, res_pad):
    import torch
    layer = _layer(i, CASES[i])
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, layer.stride, layer.pad, layer.relu, layer.pool)
    Ho = (H + 2 * layer.pad - R) // layer.stride + 1
    Wo = (W + 2 * layer.pad - S) // layer.stride + 1
    res = np.random.default_rng(100 + i).uniform(-1, 1, (N, K, Ho, Wo)).astype(np.float32)
    res_dev = torch.from_numpy(np.pad(res, ((0, 0), (0, 0), (res_pad, res_pad), (res_pad, res_pad)))).cuda()
    say("residual", res_pad, CASES[i], L.plan(N))
    xp = L.pad_input(torch.from_numpy(layer.x).cuda())
    out = L.forward_padded(xp, residual=res_dev, residual_pad=res_pad)
    torch.cuda.synchronize()
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, layer.stride, layer.pad, layer.relu, layer.pool,
                          residual=res)
    check_close(out.cpu().numpy(), ref, ab, f"residual {CASES[i]}")


@pytest.mark.parametrize("i", [0, 2, 7])
def test_misaligned_output_and_residual_match_aligned_bitwise(sp, i):
    """Output and residual tensors that start 4 bytes past an 8-byte boundary
    give the same bits as aligned ones (with even widths a lane's pixel pair
    moves with one two-dword access, which needs only 4-byte alignment; odd
    widths store element by element)."""
    import torch
    layer = _layer(i, CASES[i])
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, layer.stride, layer.pad, layer.relu, layer.pool)
    Ho, Wo = L.Ho, L.Wo
    say("misaligned out/residual", CASES[i], L.plan(N))
    xp = L.pad_input(torch.from_numpy(layer.x).cuda())
    res = np.random.default_rng(300 + i).uniform(-1, 1, (N, K, Ho, Wo)).astype(np.float32)
    n = res.size
    res_a = torch.from_numpy(res).cuda()
    res_base = torch.empty(n + 1, device="cuda")
    res_m = res_base[1:].view(N, K, Ho, Wo)
    res_m.copy_(res_a)
    out_a = torch.full((N, K, Ho, Wo), float("nan"), device="cuda")
    out_base = torch.full((n + 1,), float("nan"), device="cuda")
    out_m = out_base[1:].view(N, K, Ho, Wo)
    assert out_a.data_ptr() % 8 == 0 and out_m.data_ptr() % 8 == 4 and res_m.data_ptr() % 8 == 4
    for res_dev in (None, res_a, res_m):
        kw = {} if res_dev is None else dict(residual=res_dev, residual_pad=0)
        L.forward_padded(xp, out=out_a, **kw)
        L.forward_padded(xp, out=out_m, **kw)
        torch.cuda.synchronize()
        assert np.array_equal(out_a.cpu().numpy().view(np.uint32), out_m.cpu().numpy().view(np.uint32))


def test_residual_and_out_pad_together(sp):
    """Both options at once, on the same call: the padded output equals the
    padded residual-only output bit for bit."""
    import torch
    layer = _layer(1, CASES[1])
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, layer.pool)
    res = torch.from_numpy(np.random.default_rng(5).uniform(-1, 1, (N, K, H + 2, W + 2)).astype(np.float32)).cuda()
    say("residual + out_pad", CASES[1])
    xp = L.pad_input(torch.from_numpy(layer.x).cuda())
    a = L.forward_padded(xp, residual=res, residual_pad=1)
    b = L.forward_padded(xp, residual=res, residual_pad=1, out_pad=1)
    torch.cuda.synchronize()
    ref = np.pad(a.cpu().numpy(), ((0, 0), (0, 0), (1, 1), (1, 1)))
    assert np.array_equal(b.cpu().numpy().view(np.uint32), ref.view(np.uint32))


def test_chained_layers_skip_the_pad_pass(sp):
    """VGG-block-shaped chain: conv1 writes conv2's padded input directly
    (out_pad = conv2's pad); the result equals the unfused chain bit for bit."""
    import torch
    rng = np.random.default_rng(9)
    N, C, K, H, W = 2, 8, 8, 32, 32
    x = np.zeros((N, C, H, W), np.float32)
    x[:, :3] = rng.random((N, 3, H, W), dtype=np.float32)
    l1 = synth.random_layer(91, N, C, K, H, W, density=0.3, relu=True, pool=False)
    l2 = synth.random_layer(92, N, K, K, H, W, density=0.3, relu=True, pool=True)
    L1 = sp.SparseConvLayer(l1.w, l1.mask, l1.bias, H, W, 1, 1, True, False)
    L2 = sp.SparseConvLayer(l2.w, l2.mask, l2.bias, H, W, 1, 1, True, True)
    say("chain fused", x.shape)
    xd = torch.from_numpy(x).cuda()
    unfused = L2.run(L1.run(xd))
    y1p = L1.forward_padded(L1.pad_input(xd), out_pad=1)
    fused = L2.forward_padded(y1p)
    torch.cuda.synchronize()
    assert np.array_equal(fused.cpu().numpy().view(np.uint32), unfused.cpu().numpy().view(np.uint32))


def test_resnet_basic_block(sp):
    """relu(conv2(relu(conv1(x))) + x) with conv1 writing conv2's padded input
    and conv2 reading the shortcut from the padded block input: each stage
    against the oracle on that stage's own GPU input."""
    import torch
    rng = np.random.default_rng(12)
    N, C, H, W = 4, 16, 14, 14
    x = rng.uniform(0, 1, (N, C, H, W)).astype(np.float32)
    l1 = synth.random_layer(121, N, C, C, H, W, density=0.2, relu=True, pool=False)
    l2 = synth.random_layer(122, N, C, C, H, W, density=0.2, relu=True, pool=False)
    L1 = sp.SparseConvLayer(l1.w, l1.mask, l1.bias, H, W, 1, 1, True, False)
    L2 = sp.SparseConvLayer(l2.w, l2.mask, l2.bias, H, W, 1, 1, True, False)
    say("resnet block", x.shape)
    xp = L1.pad_input(torch.from_numpy(x).cuda())
    y1p = L1.forward_padded(xp, out_pad=1)
    y2 = L2.forward_padded(y1p, residual=xp, residual_pad=1)
    torch.cuda.synchronize()
    y1 = y1p.cpu().numpy()[:, :, 1:-1, 1:-1]
    r1, a1 = oracle.conv(x, l1.w, l1.mask, l1.bias, 1, 1, True, False)
    check_close(y1, r1, a1, "block conv1")
    r2, a2 = oracle.conv(np.ascontiguousarray(y1), l2.w, l2.mask, l2.bias, 1, 1, True, False, residual=x)
    check_close(y2.cpu().numpy(), r2, a2, "block conv2 + shortcut")


def test_row_spanning_tiles_with_residual_and_border(sp):
    """A 224x224 layer of 32 images plans row-spanning tiles with a lowered
    stream (tiles of 64*PI - 2 virtual pixels starting in any column) and
    whole-row tiles without one: with a residual read from a bordered tensor
    and a bordered output, the two launches give the same bits, and both the
    oracle's values inside an all-zero border."""
    import torch
    layer = synth.random_layer(8900, 32, 32, 64, 224, 224, density=0.2)
    N, C, H, W, K, R, S = layer.shape
    say("row-spanning tiles", layer.shape)
    rng = np.random.default_rng(8901)
    res = rng.uniform(-1, 1, (N, K, H, W)).astype(np.float32)
    resp = np.pad(res, ((0, 0), (0, 0), (1, 1), (1, 1)))
    outs = {}
    for lowered in (False, True):
        L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False, lowered=lowered)
        plan = L.plan(N)
        assert (plan["tile_pixels"] > 0) == lowered, plan
        xd = torch.from_numpy(layer.x).cuda()
        xp = L.pad_input(xd)
        out = torch.full((N, K, H + 2, W + 2), float("nan"), device="cuda")
        L.forward_padded(xp, out=out, out_pad=1, residual=torch.from_numpy(resp).cuda(), residual_pad=1)
        torch.cuda.synchronize()
        outs[lowered] = out.cpu().numpy()
    assert np.array_equal(outs[False].view(np.uint32), outs[True].view(np.uint32))
    o = outs[True]
    border = np.ones(o.shape[2:], bool)
    border[1:-1, 1:-1] = False
    assert np.all(o[:, :, border].view(np.uint32) == 0)
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 1, 1, True, False, residual=res)
    check_close(o[:, :, 1:-1, 1:-1], ref, ab, "row-spanning tiles")
