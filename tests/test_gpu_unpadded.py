"""GPU tests of SPCONV_UNPADDED_INPUT: the kernels read the unpadded NCHW
input and form the zero border in LDS (the pad step fused into the
convolution). Every stored output reads only staged rows and columns that hold
the same values as with a padded input, and the arithmetic is unchanged, so
the outputs must equal the padded path's bit for bit — on every stride-1 case
and kernel variant of the parity suite, with the epilogue options, and on the
dense path. Plans of the any-stride kernel reject the flag; the layer object
then pads first. Every case prints its name and plan before touching the GPU.
"""
import numpy as np
import pytest

import oracle
from paper_2005_04091_amd import synth
import test_gpu_parity as tp

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sp():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2005_04091_amd import spconv
    return spconv


def say(*a):
    print("[case]", *a, flush=True)


def bitwise(a, b, what):
    a, b = a.cpu().numpy(), b.cpu().numpy()
    assert a.shape == b.shape, (a.shape, b.shape)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), f"{what}: unpadded input differs from padded"


def _both(sp, L, x, **kw):
    import torch
    xd = torch.from_numpy(x).cuda()
    fused = L.forward(xd, pad_in_kernel=True, **kw)
    plain = L.forward_padded(L.pad_input(xd), **kw)
    torch.cuda.synchronize()
    return fused, plain


STRIDE1_CASES = [c for c in tp.SWEEP if c[7] == 1]


@pytest.mark.parametrize("i", range(len(STRIDE1_CASES)))
def test_unpadded_equals_padded_cases(sp, i):
    N, C, K, H, W, R, S, stride, pad, d, relu, pool, bias, skew = STRIDE1_CASES[i]
    layer = synth.random_layer(6100 + i, N, C, K, H, W, R, S, stride, pad, d, relu, pool, bias, skew)
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, stride, pad, relu, pool)
    say("unpadded case", STRIDE1_CASES[i], L.plan(N))
    fused, plain = _both(sp, L, layer.x)
    bitwise(fused, plain, str(STRIDE1_CASES[i]))


@pytest.mark.parametrize("case", tp.VARIANTS, ids=[v[0] for v in tp.VARIANTS])
def test_unpadded_equals_padded_variants(sp, case):
    name, N, C, K, H, pool, skew, expect = case
    layer = synth.random_layer(4242, N, C, K, H, H, density=0.3, pool=pool, skew=skew)
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, H, 1, 1, True, pool)
    plan = L.plan(N)
    say("unpadded variant", name, plan)
    assert (plan["pixels_per_lane"], plan["images_per_group"], plan["channels_per_wave"]) == expect
    assert L.can_pad_in_kernel(N)
    fused, plain = _both(sp, L, layer.x)
    bitwise(fused, plain, name)


@pytest.mark.parametrize("opt", ["out_pad", "residual", "both"])
def test_unpadded_with_epilogue_options(sp, opt):
    import torch
    layer = synth.random_layer(6200, 3, 12, 20, 23, 19, 3, 3, 1, 1, 0.3, True, False, True, False)
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False)
    kw = {}
    if opt in ("out_pad", "both"):
        kw["out_pad"] = 1
    if opt in ("residual", "both"):
        res = np.random.default_rng(1).uniform(-1, 1, (N, K, H + 2, W + 2)).astype(np.float32)
        kw.update(residual=torch.from_numpy(res).cuda(), residual_pad=1)
    say("unpadded epilogue", opt, L.plan(N))
    fused, plain = _both(sp, L, layer.x, **kw)
    bitwise(fused, plain, opt)


@pytest.mark.parametrize("i", [0, 1, 4, 6, 7, 11])
def test_unpadded_dense(sp, i):
    from test_gpu_dense import CASES, _layer
    layer = _layer(i)
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, layer.pad, True, layer.pool, path="dense")
    say("unpadded dense", CASES[i], L.plan(N))
    fused, plain = _both(sp, L, layer.x)
    bitwise(fused, plain, f"dense {CASES[i]}")


def test_stride2_pads_first_and_flag_is_rejected(sp):
    import torch
    layer = synth.random_layer(6300, 2, 5, 7, 9, 8, 3, 3, 2, 1, 0.4, True, False, True, False)
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 2, 1, True, False)
    say("unpadded stride 2", L.plan(N))
    assert not L.can_pad_in_kernel(N) and not L.pads_in_kernel(N)
    x = torch.from_numpy(layer.x).cuda()
    with pytest.raises(sp.SpconvError):
        L.forward_padded(x, _extra_flags=sp.SPCONV_UNPADDED_INPUT)
    with pytest.raises(ValueError):
        L.forward(x, pad_in_kernel=True)
    out = L.forward(x)
    torch.cuda.synchronize()
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 2, 1, True, False)
    tp.check_close(out.cpu().numpy(), ref, ab, "stride 2")


def test_unpadded_resnet_full_size(sp):
    """The benchmarked ResNet layer through the fused-pad forward, whole output
    tensor against the oracle."""
    import torch
    layer = synth.make_layer("resnet")
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False, path="auto", N=N)
    say("unpadded resnet", L.path, L.plan(N))
    out = L.forward(torch.from_numpy(layer.x).cuda(), pad_in_kernel=True)
    torch.cuda.synchronize()
    ref, ab = oracle.conv(layer.x, layer.w, layer.mask, layer.bias, 1, 1, True, False)
    tp.check_close(out.cpu().numpy(), ref, ab, "unpadded resnet")


def test_resnet_block_without_pad_passes_bitwise(sp):
    """A ResNet basic block as two launches on unpadded tensors (the shortcut
    is the block input itself) equals the block chained through a
    zero-bordered output, bit for bit."""
    import torch
    x, l1, l2 = synth.make_resnet_block()
    x = x[:4].copy()
    N, C, H, W = x.shape
    L1 = sp.SparseConvLayer(l1.w, l1.mask, l1.bias, H, W, 1, 1, True, False)
    L2 = sp.SparseConvLayer(l2.w, l2.mask, l2.bias, H, W, 1, 1, True, False)
    say("resnet block unpadded", L1.plan(N), L2.plan(N))
    xd = torch.from_numpy(x).cuda()
    y2 = L2.forward(L1.forward(xd, pad_in_kernel=True), residual=xd, residual_pad=0, pad_in_kernel=True)
    xp = L1.pad_input(xd)
    y1p = L1.forward_padded(xp, out_pad=1)
    z2 = L2.forward_padded(y1p, residual=xp, residual_pad=1)
    torch.cuda.synchronize()
    bitwise(y2, z2, "resnet block")
