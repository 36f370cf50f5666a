"""GPU tests of the resize prologue (spconv_resize_pad_input) and of the
Resize-Conv-ReLU-Maxpool block it feeds.

Resize: bilinear with pixel centres aligned, written with a zero border into
the padded layout. Tolerance, derived from the kernel's arithmetic: each of the
three fp32 interpolations a + t*(b - a) adds at most about 5 ulp of the
largest tap magnitude M (one rounding each for b - a, t, the product and the
sum, the first two scaled by |b - a| <= 2M), and the outer one carries the
inner errors through a convex combination, so |gpu - exact| <= 10 * 2^-24 * M
~= 6e-7 * M; the tests allow 1e-6 * max|x|. The border must be +0.0 bit for
bit, and an unchanged size must reproduce spconv_pad_input bit for bit.

Block: the convolution of the GPU-resized input is checked against the oracle
on that same fp32 input (the layer tolerance 1e-5 * sum|w*x| + 1e-6), and the
whole block against the oracle's resize followed by its convolution, with the
resize tolerance carried through the filter: + 2e-6 * M * sum_j |w_kj| (ReLU and
max-pool do not enlarge a difference). Every case prints its name and shape
before touching the GPU.
"""
import numpy as np
import pytest

import oracle
from paper_2005_04091_amd import synth

pytestmark = pytest.mark.gpu

RESIZE_TOL = 1e-6
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


# N, C, Hin, Win, H, W, pad: up and down, non-integer ratios, one-pixel source
# and output, narrow and wide planes, several planes per workgroup (flat
# variant); the last two take the row variant: a padded plane whose tap tables
# exceed the LDS budget (split into row bands), and 1x1 outputs of sources too
# large for one workgroup's 32-bit source offsets.
CASES = [
    (1, 2, 7, 9, 5, 13, 1),
    (2, 3, 42, 42, 28, 28, 1),
    (2, 1, 1, 1, 3, 4, 2),
    (1, 1, 3, 3, 1, 1, 0),
    (1, 1, 9, 300, 5, 270, 0),
    (1, 1, 5, 5, 3, 200, 3),
    (1, 1, 100, 100, 130, 150, 2),
    (3, 2, 17, 4, 64, 61, 1),
    (4, 3, 224, 224, 112, 112, 1),
    (64, 40, 56, 56, 28, 28, 1),
    (5, 7, 3, 2, 1, 1, 0),
    (1, 1, 6, 4100, 10, 4100, 1),
    (2, 2, 1100, 1100, 1, 1, 0),
]


def _src(seed, shape):
    return np.random.default_rng(seed).uniform(-1, 1, shape).astype(np.float32)


def check_resize(got_padded, x, H, W, pad, what):
    ref, _ = oracle.resize(x, H, W)
    inner = got_padded[:, :, pad:pad + H, pad:pad + W].astype(np.float64)
    err = np.abs(inner - ref)
    tol = RESIZE_TOL * float(np.abs(x).max())
    assert err.max() <= tol, f"{what}: max err {err.max():.3e} > {tol:.3e}"
    border = got_padded.copy()
    border[:, :, pad:pad + H, pad:pad + W] = 0.0
    assert not border.view(np.uint32).any(), f"{what}: border is not +0.0"


@pytest.mark.parametrize("i", range(len(CASES)))
def test_resize_against_oracle(sp, i):
    import torch
    N, C, Hin, Win, H, W, pad = CASES[i]
    x = _src(300 + i, (N, C, Hin, Win))
    say("resize", CASES[i])
    xd = torch.from_numpy(x).cuda()
    out = torch.full((N, C, H + 2 * pad, W + 2 * pad), float("nan"), device="cuda")
    sp.spconv_resize_pad_input(xd, H, W, pad, out=out)
    torch.cuda.synchronize()
    check_resize(out.cpu().numpy(), x, H, W, pad, f"resize {CASES[i]}")


@pytest.mark.parametrize("shape", [(2, 3, 20, 30, 1), (1, 2, 5, 270, 2), (3, 1, 56, 56, 1), (1, 1, 1, 1, 0)])
def test_unchanged_size_is_the_pad_pass_bitwise(sp, shape):
    import torch
    N, C, H, W, pad = shape
    x = _src(17, (N, C, H, W))
    say("resize identity", shape)
    xd = torch.from_numpy(x).cuda()
    a = sp.spconv_resize_pad_input(xd, H, W, pad)
    b = sp.spconv_pad_input(xd, pad)
    torch.cuda.synchronize()
    assert np.array_equal(a.cpu().numpy().view(np.uint32), b.cpu().numpy().view(np.uint32))


def test_second_call_overwrites_every_element(sp):
    """A smaller call after a larger one on the same buffer: every element of
    the smaller padded tensor is rewritten (no stale values, border included)."""
    import torch
    big = _src(5, (2, 2, 30, 30))
    small = _src(6, (1, 2, 9, 7))
    say("resize reuse")
    buf = torch.full((2 * 2 * 34 * 34,), float("nan"), device="cuda")
    sp.spconv_resize_pad_input(torch.from_numpy(big).cuda(), 32, 32, 1, out=buf.view(2, 2, 34, 34))
    out = buf[:1 * 2 * 13 * 11].view(1, 2, 13, 11)
    sp.spconv_resize_pad_input(torch.from_numpy(small).cuda(), 11, 9, 1, out=out)
    torch.cuda.synchronize()
    check_resize(out.cpu().numpy(), small, 11, 9, 1, "resize reuse")


def _block_tol(layer, ab, M):
    wsum = np.abs(layer.w.astype(np.float64)).reshape(layer.w.shape[0], -1).sum(axis=1)
    return REL_TOL * ab + ABS_TOL + 2.0 * RESIZE_TOL * M * wsum[None, :, None, None]


@pytest.mark.parametrize("case", [(2, 6, 10, 23, 17, 14, 12, 0.3), (1, 16, 16, 9, 9, 20, 24, 0.2),
                                  (3, 5, 7, 30, 44, 30, 44, 0.4)])
def test_resize_conv_relu_maxpool_block(sp, case):
    """Stage by stage and end to end against the oracle."""
    import torch
    N, C, K, Hin, Win, H, W, d = case
    layer = synth.random_layer(900 + Hin, N, C, K, H, W, 3, 3, 1, 1, d, True, True, True, False)
    src = np.random.default_rng(Hin).random((N, C, Hin, Win), dtype=np.float32)
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, True)
    say("resize block", case, L.plan(N))
    xp = L.resize_pad_input(torch.from_numpy(src).cuda())
    out = L.forward_padded(xp)
    torch.cuda.synchronize()
    xp_h = xp.cpu().numpy()
    got = out.cpu().numpy().astype(np.float64)
    check_resize(xp_h, src, H, W, 1, f"block resize {case}")
    ref, ab = oracle.conv(xp_h[:, :, 1:-1, 1:-1], layer.w, layer.mask, layer.bias, 1, 1, True, True)
    err = np.abs(got - ref)
    assert (err <= REL_TOL * ab + ABS_TOL).all(), f"conv on the resized input: max err {err.max():.3e}"
    rs, _ = oracle.resize(src, H, W)
    ref2, ab2 = oracle.conv(rs.astype(np.float32), layer.w, layer.mask, layer.bias, 1, 1, True, True)
    err2 = np.abs(got - ref2)
    assert (err2 <= _block_tol(layer, ab2, float(np.abs(src).max()))).all(), f"end to end: max err {err2.max():.3e}"


def test_resize_block_full_size(sp):
    """The benchmarked block at full size (32 x 128 x 42x42 -> 28x28, conv,
    ReLU, 2x2 max-pool), in the launch configuration the benchmark times: the
    whole resized tensor against the oracle, and the whole block output end
    to end."""
    import torch
    src, layer = synth.make_resize_block()
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, True)
    say("resize block full size", (N, C, src.shape[2], src.shape[3], H, W), L.plan(N))
    xp = L.resize_pad_input(torch.from_numpy(src).cuda())
    out = L.forward_padded(xp)
    torch.cuda.synchronize()
    check_resize(xp.cpu().numpy(), src, H, W, 1, "full-size resize")
    got = out.cpu().numpy().astype(np.float64)
    rs, _ = oracle.resize(src, H, W)
    ref, ab = oracle.conv(rs.astype(np.float32), layer.w, layer.mask, layer.bias, 1, 1, True, True)
    err = np.abs(got - ref)
    tol = _block_tol(layer, ab, float(np.abs(src).max()))
    assert (err <= tol).all(), f"end to end: {int((err > tol).sum())} outputs out of bound, max err {err.max():.3e}"
