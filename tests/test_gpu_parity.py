"""GPU parity: the HIP path against the CPU oracle, element by element.

Acceptance per output element: |gpu - oracle| <= 1e-5 * A + 1e-6, where A is the
oracle's sum of |w * x| over the terms of that output (its max over the window for
pooled outputs). Index work (padding) is compared bit for bit. Every case prints
its name and shape before touching the GPU.
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
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite output"
    err = np.abs(gpu - ref)
    tol = REL_TOL * ab + ABS_TOL
    bad = err > tol
    if bad.any():
        i = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outputs out of tolerance; worst at {i}: "
                             f"gpu={gpu[i]!r} oracle={ref[i]!r} A={ab[i]!r}")


def run_layer(sp, layer, stream=None):
    import torch
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, layer.stride, layer.pad, layer.relu, layer.pool)
    x = torch.from_numpy(layer.x).cuda()
    out = L.run(x, stream=stream)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def oracle_layer(layer, pairs=None):
    return oracle.conv(layer.x, layer.w, layer.mask, layer.bias, layer.stride, layer.pad, layer.relu, layer.pool,
                       pairs=pairs)


# ---------------------------------------------------------------------------
# Padded input: bit exact against numpy.pad
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("shape,pad", [((1, 1, 1, 1), 0), ((1, 1, 1, 1), 3), ((2, 3, 5, 7), 1), ((3, 2, 17, 9), 2),
                                       ((2, 4, 56, 56), 1), ((1, 3, 33, 65), 0), ((4, 5, 13, 300), 4)])
def test_pad_bit_exact(sp, shape, pad):
    import torch
    say("pad", shape, pad)
    rng = np.random.default_rng(sum(shape) + pad)
    x = rng.uniform(-1, 1, shape).astype(np.float32)
    x.reshape(-1)[::7] = -0.0
    xp = sp.spconv_pad_input(torch.from_numpy(x).cuda(), pad)
    torch.cuda.synchronize()
    ref = oracle.pad(x, pad)
    assert np.array_equal(xp.cpu().numpy().view(np.uint32), ref.view(np.uint32))


def test_pad_unaligned_output_and_guards(sp):
    """An output that starts 4 bytes past a 16-byte boundary (the kernel's
    scalar-store variant), between NaN guard words that must survive."""
    import torch
    x = np.random.default_rng(8).uniform(-1, 1, (3, 2, 11, 13)).astype(np.float32)
    ref = oracle.pad(x, 2)
    buf = torch.full((ref.size + 9,), float("nan"), dtype=torch.float32, device="cuda")
    out = buf[1:1 + ref.size].view(ref.shape)
    say("pad unaligned")
    sp.spconv_pad_input(torch.from_numpy(x).cuda(), 2, out=out)
    torch.cuda.synchronize()
    b = buf.cpu().numpy()
    assert np.isnan(b[0]) and np.isnan(b[1 + ref.size:]).all()
    assert np.array_equal(b[1:1 + ref.size].view(np.uint32), ref.reshape(-1).view(np.uint32))


# ---------------------------------------------------------------------------
# Forward: small shapes spanning tiles, ragged tails and the degenerate cases
# ---------------------------------------------------------------------------

SWEEP = [
    # N, C, K, H, W, R, S, stride, pad, density, relu, pool, bias, skew
    (1, 16, 16, 16, 16, 3, 3, 1, 1, 0.2, True, False, True, False),
    (2, 3, 5, 7, 9, 3, 3, 1, 1, 0.5, True, False, True, False),      # odd, H != W, K ragged
    (3, 4, 6, 11, 13, 3, 3, 1, 0, 0.3, False, False, True, False),   # pad 0, N ragged vs images per group
    (2, 5, 7, 9, 8, 3, 3, 2, 1, 0.4, True, False, True, False),      # stride 2
    (2, 5, 3, 10, 12, 3, 3, 2, 1, 0.4, True, True, True, False),     # stride 2 + pool
    (1, 6, 9, 12, 10, 5, 5, 1, 2, 0.3, True, False, False, False),   # 5x5, no bias
    (2, 4, 8, 9, 15, 3, 1, 1, 1, 0.5, True, False, True, False),     # 3x1
    (2, 4, 8, 9, 15, 1, 3, 1, 1, 0.5, True, False, True, False),     # 1x3 (pad makes Ho > H)
    (2, 8, 12, 14, 14, 1, 1, 1, 0, 0.5, True, False, True, False),   # 1x1
    (2, 3, 4, 8, 8, 2, 2, 1, 0, 0.6, True, True, True, False),       # 2x2, pool
    (2, 8, 10, 13, 11, 3, 3, 1, 1, 0.3, True, True, True, False),    # pool with odd Ho/Wo (floor)
    (1, 2, 3, 6, 6, 3, 3, 1, 1, 0.0, True, False, True, False),      # density 0: act(bias)
    (2, 3, 5, 6, 7, 3, 3, 1, 1, 1.0, False, False, True, False),     # density 1, no ReLU
    (2, 200, 9, 10, 10, 3, 3, 1, 1, 0.1, True, False, True, False),  # C spans several LDS chunks
    (2, 64, 33, 20, 20, 3, 3, 1, 1, 0.2, True, False, True, True),   # skewed rows, K ragged vs 8
    (1, 8, 16, 60, 64, 3, 3, 1, 1, 0.2, True, False, True, False),   # several spatial tiles
    (2, 8, 16, 61, 70, 3, 3, 1, 1, 0.2, True, True, True, False),    # several tiles + pool, odd Ho
    (1, 4, 4, 5, 300, 3, 3, 1, 1, 0.3, True, False, True, False),    # wide rows (tile < one row pair)
    (5, 16, 20, 14, 14, 3, 3, 1, 1, 0.05, True, False, True, False), # small planes, several images per group
    (1, 1, 1, 1, 1, 1, 1, 1, 0, 1.0, False, False, True, False),     # 1x1x1x1
    (2, 3, 4, 2, 2, 3, 3, 1, 1, 0.7, True, True, True, False),       # tiny pooled output (1x1)
]


@pytest.mark.parametrize("case", SWEEP, ids=[f"sweep{i}" for i in range(len(SWEEP))])
def test_forward_sweep(sp, case):
    N, C, K, H, W, R, S, stride, pad, d, relu, pool, bias, skew = case
    layer = synth.random_layer(1000 + hash(case) % 1000, N, C, K, H, W, R, S, stride, pad, d, relu, pool, bias, skew)
    say("sweep", case)
    gpu = run_layer(sp, layer)
    ref, ab = oracle_layer(layer)
    check_close(gpu, ref, ab, f"sweep {case}")


def test_single_row_holds_every_nonzero(sp):
    """Maximal skew: one output channel has every tap, the others none."""
    layer = synth.random_layer(77, 2, 32, 12, 18, 18, 3, 3, 1, 1, 1.0, True, False, True)
    layer.mask[:] = 0
    layer.mask[5] = 1
    layer.w = np.where(layer.mask != 0, np.random.default_rng(1).uniform(-1, 1, layer.w.shape), 0).astype(np.float32)
    say("single-row skew")
    gpu = run_layer(sp, layer)
    ref, ab = oracle_layer(layer)
    check_close(gpu, ref, ab, "single row")


def test_identity_filter_bitwise(sp):
    """One 1.0 per row at (c = k, centre tap): output == input bit for bit, and
    with pooling the 2x2 block max of the input."""
    rng = np.random.default_rng(3)
    N, C, H, W = 3, 24, 30, 27
    x = rng.random((N, C, H, W), dtype=np.float32)
    w = np.zeros((C, C, 3, 3), np.float32)
    for k in range(C):
        w[k, k, 1, 1] = 1.0
    for pool in (False, True):
        layer = synth.Layer("identity", x, w, (w != 0).astype(np.uint8), None, 1, 1, True, pool)
        say("identity", pool)
        gpu = run_layer(sp, layer)
        ref = x if not pool else x[:, :, :H // 2 * 2, :W // 2 * 2].reshape(N, C, H // 2, 2, W // 2, 2).max(axis=(3, 5))
        assert np.array_equal(gpu.view(np.uint32), ref.view(np.uint32))


# ---------------------------------------------------------------------------
# The named layers at full size, in the launch configuration the benchmark uses
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny", "resnet", "conv_pool", "narrow_d0.05", "narrow_d0.2", "narrow_d0.5"])
def test_named_layer_full(sp, name):
    layer = synth.make_layer(name)
    say("layer", name, layer.shape)
    gpu = run_layer(sp, layer)
    ref, ab = oracle_layer(layer)
    check_close(gpu, ref, ab, name)


@pytest.mark.parametrize("which", [1, 2])
def test_vgg_layers_full_size(sp, which):
    """Each VGG-block layer at 32 x 64 x 224 x 224, the whole output tensor
    against the oracle."""
    _, l1, l2 = synth.make_vgg_block()
    layer = l1 if which == 1 else l2
    say("vgg layer", which, layer.shape)
    gpu = run_layer(sp, layer)
    ref, ab = oracle_layer(layer)
    check_close(gpu, ref, ab, f"vgg layer {which}")


def _chain_check(sp, x, l1, l2):
    """Chained layers on the GPU (layer 2 reads layer 1's GPU output) against the
    oracle chain (layer 2 applied to layer 1's oracle output rounded to fp32),
    image by image over every output. The bound adds, to layer 2's own
    tolerance, the propagated layer-1 error sum |w2| * (1e-5*A1 + 1e-6 + |y1| *
    2^-24), evaluated by the oracle itself (ReLU and max-pool are 1-Lipschitz)."""
    import torch
    N, C, H, W, K, R, S = l1.shape
    L1 = sp.SparseConvLayer(l1.w, l1.mask, l1.bias, H, W, 1, 1, l1.relu, l1.pool)
    L2 = sp.SparseConvLayer(l2.w, l2.mask, l2.bias, H, W, 1, 1, l2.relu, l2.pool)
    y1 = L1.run(torch.from_numpy(x).cuda())
    y2 = L2.run(y1)
    torch.cuda.synchronize()
    y2 = y2.cpu().numpy()
    for n in range(N):
        xo = x[n:n + 1]
        r1, a1 = oracle.conv(xo, l1.w, l1.mask, l1.bias, 1, 1, l1.relu, l1.pool)
        x2 = r1.astype(np.float32)
        r2, a2 = oracle.conv(x2, l2.w, l2.mask, l2.bias, 1, 1, l2.relu, l2.pool)
        delta = (REL_TOL * a1 + ABS_TOL + np.abs(r1) * 2.0 ** -24) * (1 + 1e-6)
        prop, _ = oracle.conv(delta.astype(np.float32), np.abs(l2.w), l2.mask, None, 1, 1, False, l2.pool)
        err = np.abs(y2[n:n + 1].astype(np.float64) - r2)
        tol = REL_TOL * a2 + ABS_TOL + prop
        assert np.all(err <= tol), f"chain image {n}: {(err > tol).sum()} outputs out of bound"


def test_chain_small(sp):
    """Two chained layers at a size the oracle covers whole (VGG-block shape, scaled)."""
    rng = np.random.default_rng(9)
    N, C, K, H, W = 2, 8, 8, 32, 32
    x = np.zeros((N, C, H, W), np.float32)
    x[:, :3] = rng.random((N, 3, H, W), dtype=np.float32)
    l1 = synth.random_layer(91, N, C, K, H, W, density=0.3, relu=True, pool=False)
    l2 = synth.random_layer(92, N, K, K, H, W, density=0.3, relu=True, pool=True)
    say("chain small")
    _chain_check(sp, x, l1, l2)


def test_vgg_block_chain_full_size(sp):
    """The VGG-style block as the benchmark runs it (32 images, chained), every
    output of every image against the oracle chain."""
    x, l1, l2 = synth.make_vgg_block()
    say("vgg chain", x.shape)
    _chain_check(sp, x, l1, l2)


# ---------------------------------------------------------------------------
# Every stride-1 kernel variant the planner picks: pixels per lane x images
# per workgroup x channels per wave, pooled or not, one or several LDS chunks,
# CSR rows with more than a window (128 entries) in one chunk, channel tiles
# and image groups cut short at the end. The planner's pick is asserted, so a
# change of the planner that leaves a variant untested fails here.
# ---------------------------------------------------------------------------

VARIANTS = [
    # name, N, C, K, H(=W), pool, skewed rows, expected (PI, IPW, RPW)
    ("ipw1_rpw2", 8, 3, 520, 12, False, True, (4, 1, 2)),
    ("ipw1_rpw2_pool", 4, 16, 1040, 12, True, True, (4, 1, 2)),
    ("ipw1_rpw4", 16, 3, 520, 12, False, True, (4, 1, 4)),
    ("ipw2_rpw1", 8, 3, 520, 2, False, False, (2, 2, 1)),
    ("ipw2_rpw1_pool", 8, 3, 520, 2, True, False, (2, 2, 1)),
    ("ipw2_rpw2", 16, 3, 520, 2, False, True, (2, 2, 2)),
    ("ipw2_rpw2_pool", 8, 16, 1040, 2, True, True, (2, 2, 2)),
    ("ipw2_rpw4", 32, 3, 520, 2, False, True, (2, 2, 4)),
    ("ipw4_rpw2_ragged_n", 31, 3, 520, 2, False, False, (2, 4, 2)),
    ("ipw4_rpw4", 64, 3, 520, 2, False, False, (2, 4, 4)),
    ("ipw4_rpw4_pool", 32, 3, 1040, 2, True, True, (2, 4, 4)),
    ("ipw2_rpw2_chunks_overflow", 16, 700, 520, 2, False, True, (2, 2, 2)),
    ("ipw2_rpw1_chunks", 32, 700, 520, 2, False, False, (2, 2, 1)),
    ("ipw1_rpw4_chunks_overflow", 16, 250, 520, 12, False, True, (4, 1, 4)),
    ("ipw1_rpw2_pool_chunks_overflow", 8, 250, 520, 12, True, True, (4, 1, 2)),
    ("ipw4_rpw1_pool", 16, 3, 520, 2, True, False, (2, 4, 1)),
    ("ipw4_rpw2_pool", 32, 3, 520, 2, True, False, (2, 4, 2)),
    # more work items than CUs, the last round partly filled (495 items): the
    # lowered kernel runs several work items per workgroup
    ("ipw1_rpw1_495_items", 33, 3, 48, 64, False, False, (14, 1, 1)),
    ("ipw1_rpw1_pool_495_items", 33, 3, 48, 56, True, False, (12, 1, 1)),
    # ... with the pooled staging of pair maxima in the last chunk's buffer,
    # so the next tile's first chunk is copied during the last one (504 items)
    ("ipw1_rpw1_pool_pairs_504_items", 9, 32, 16, 224, True, False, (16, 1, 1)),
]


@pytest.mark.parametrize("case", VARIANTS, ids=[v[0] for v in VARIANTS])
def test_kernel_variant(sp, case):
    import torch
    name, N, C, K, H, pool, skew, expect = case
    layer = synth.random_layer(4242, N, C, K, H, H, density=0.3, pool=pool, skew=skew)
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, H, 1, 1, True, pool)
    plan = L.plan(N)
    say("variant", name, layer.shape, plan)
    assert (plan["pixels_per_lane"], plan["images_per_group"], plan["channels_per_wave"]) == expect
    if "chunks" in name:
        assert plan["chunks"] >= 2, "the variant must span several LDS chunks"
    if "items" in name:
        assert plan["workgroups"] > plan["launch_workgroups"] == 256 and plan["workgroups"] % 256
    out = L.run(torch.from_numpy(layer.x).cuda())
    torch.cuda.synchronize()
    ref, ab = oracle_layer(layer)
    check_close(out.cpu().numpy(), ref, ab, name)


def test_plan_hint_changes_tiling_not_results(sp):
    """Without the max_row_nnz hint the planner takes another tiling for a
    skewed filter; every output still sums its row's entries in CSR order, so
    both runs agree bit for bit (and with the oracle)."""
    import torch
    layer = synth.random_layer(4343, 32, 16, 256, 14, 14, density=0.3, skew=True)
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False)
    x = torch.from_numpy(layer.x).cuda()
    hinted = L.plan(N)
    a = L.run(x).cpu().numpy()
    L.csr.max_row_nnz = 0
    blind = L.plan(N)
    say("hint", hinted, blind)
    b = L.run(x).cpu().numpy()
    assert hinted["channels_per_wave"] != blind["channels_per_wave"] or \
        hinted["pixels_per_lane"] != blind["pixels_per_lane"]
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    ref, ab = oracle_layer(layer)
    check_close(a, ref, ab, "hinted")


# ---------------------------------------------------------------------------
# Robustness
# ---------------------------------------------------------------------------

def test_guard_bands_and_full_coverage(sp):
    """Output written exactly once per element: a NaN-filled buffer with guard
    bands on both sides keeps its guards and has no NaN left inside."""
    import torch
    for pool in (False, True):
        layer = synth.random_layer(55, 3, 12, 10, 19, 23, density=0.3, pool=pool)
        N, C, H, W, K, R, S = layer.shape
        L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, pool)
        n_out = N * K * L.Ho * L.Wo
        guard = 4096
        buf = torch.full((n_out + 2 * guard,), float("nan"), dtype=torch.float32, device="cuda")
        buf[:guard] = 7.0
        buf[-guard:] = -7.0
        out = buf[guard:guard + n_out].view(N, K, L.Ho, L.Wo)
        say("guard", pool)
        L.run(torch.from_numpy(layer.x).cuda(), out=out)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.all(b[:guard] == 7.0) and np.all(b[-guard:] == -7.0)
        assert not np.isnan(b[guard:guard + n_out]).any()


def test_deterministic_and_stream_ordered(sp):
    """Repeated runs are bit-identical, also on a non-default stream."""
    import torch
    layer = synth.make_layer("tiny")
    say("determinism")
    a = run_layer(sp, layer)
    b = run_layer(sp, layer)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        c = run_layer(sp, layer, stream=s)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(a.view(np.uint32), c.view(np.uint32))


def test_stream_argument_outside_a_stream_context(sp):
    """run(stream=s) with another stream current: the temporaries and the
    output belong to s, and the result equals the default-stream run."""
    import torch
    layer = synth.random_layer(71, 4, 16, 24, 30, 30, density=0.3)
    N, C, H, W, K, R, S = layer.shape
    L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, False)
    x = torch.from_numpy(layer.x).cuda()
    say("stream argument")
    a = L.run(x)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    outs = [L.run(x, stream=s) for _ in range(4)]  # each call's padded temporary is freed on return
    s.synchronize()
    for o in outs:
        assert np.array_equal(a.cpu().numpy().view(np.uint32), o.cpu().numpy().view(np.uint32))


def test_two_host_threads_two_streams(sp):
    """Two host threads, each with its own stream, launching the same kernel
    instance on layers of different shapes (different dynamic LDS sizes, both
    above the default 64 KiB limit) repeatedly at the same time: every result
    equals its serial run bit for bit."""
    import threading
    import torch
    layers = [synth.random_layer(83, 4, 24, 40, 56, 56, density=0.2),
              synth.random_layer(85, 4, 40, 40, 56, 56, density=0.2)]
    objs, xs, serial = [], [], []
    for layer in layers:
        N, C, H, W, K, R, S = layer.shape
        L = sp.SparseConvLayer(layer.w, layer.mask, layer.bias, H, W, 1, 1, True, layer.pool)
        x = torch.from_numpy(layer.x).cuda()
        objs.append(L)
        xs.append(x)
        serial.append(L.run(x).cpu().numpy())
    plans = [L.plan(int(x.shape[0])) for L, x in zip(objs, xs)]
    say("two threads", plans)
    inst = [(p["pixels_per_lane"], p["images_per_group"], p["channels_per_wave"]) for p in plans]
    assert inst[0] == inst[1] and plans[0]["lds_bytes"] != plans[1]["lds_bytes"]
    assert min(p["lds_bytes"] for p in plans) > 65536
    results = [[], []]
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            for _ in range(20):
                results[i].append(objs[i].run(xs[i], stream=s))
            s.synchronize()
        except Exception as e:  # reported by the main thread
            errors.append(e)

    ts = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errors, errors
    for i in range(2):
        assert len(results[i]) == 20
        for o in results[i]:
            assert np.array_equal(o.cpu().numpy().view(np.uint32), serial[i].view(np.uint32))
    ref, ab = oracle_layer(layers[1])
    check_close(serial[1], ref, ab, "two threads, layer 2")
