"""CPU tests of the dense path's host side: the packed filter layout (bit
exact against an independent numpy packing), its size, argument checks of the
dense forward call (no GPU work is queued: every call is invalid), and the
path dispatcher."""
import ctypes

import numpy as np
import pytest

from paper_2005_04091_amd import synth


@pytest.fixture(scope="module")
def sp():
    from paper_2005_04091_amd import spconv
    return spconv


def kp_of(K):
    nw = min(4, -(-K // 32))
    return -(-K // (32 * nw)) * 32 * nw


def numpy_pack(w, mask):
    K, C, R, S = w.shape
    keep = (mask != 0) if mask is not None else (w != 0)
    wk = np.where(keep, w, np.float32(0)).astype(np.float32)
    Kp, cp = kp_of(K), -(-C // 2)
    full = np.zeros((Kp, 2 * cp, R * S), np.float32)
    full[:K, :C] = wk.reshape(K, C, R * S)
    # [cp][t][k][h] <- full[k][2cp+h][t]
    return np.ascontiguousarray(full.reshape(Kp, cp, 2, R * S).transpose(1, 3, 0, 2)).reshape(-1)


@pytest.mark.parametrize("shape", [(8, 4, 3, 3), (33, 5, 3, 3), (130, 7, 1, 1), (256, 3, 3, 3), (4, 1, 3, 3),
                                   (160, 9, 1, 1), (64, 64, 3, 3)])
@pytest.mark.parametrize("use_mask", [False, True])
def test_pack_dense_matches_numpy_bitwise(sp, shape, use_mask):
    K, C, R, S = shape
    layer = synth.random_layer(sum(shape), 1, C, K, 4, 4, R, S, 1, 1 if R == 3 else 0, 0.3, True, False, True, False)
    w = layer.w.copy()
    mask = layer.mask if use_mask else None
    if use_mask:
        w.flat[np.flatnonzero(layer.mask)[:3]] = 0.0   # explicit zeros stay (as zeros)
        w.flat[np.flatnonzero(layer.mask == 0)[:3]] = 7.0  # masked-out values are dropped
    else:
        w.flat[:2] = -0.0
    got = sp.spconv_pack_dense(w, mask)
    ref = numpy_pack(w, mask)
    assert got.size == sp.spconv_dense_size(K, C, R, S) == ref.size
    assert np.array_equal(np.where(got == 0, 0, got).view(np.uint32), np.where(ref == 0, 0, ref).view(np.uint32))


def test_dense_size_and_capacity(sp):
    assert sp.spconv_dense_size(256, 256, 3, 3) == 128 * 9 * 256 * 2
    assert sp.spconv_dense_size(33, 5, 3, 3) == 3 * 9 * 64 * 2
    assert sp.spconv_dense_size(130, 7, 1, 1) == 4 * 1 * 256 * 2
    lib = sp._lib
    w = np.ones((8, 4, 3, 3), np.float32)
    buf = np.zeros(sp.spconv_dense_size(8, 4, 3, 3), np.float32)
    assert lib.spconv_pack_dense(w.ctypes.data, None, 8, 4, 3, 3, buf.ctypes.data, buf.size - 1) == sp.SPCONV_ECAPACITY
    assert not buf.any()
    assert lib.spconv_pack_dense(None, None, 8, 4, 3, 3, buf.ctypes.data, buf.size) == sp.SPCONV_EINVAL
    assert lib.spconv_pack_dense(w.ctypes.data, None, 8, 4, 3, 3, None, buf.size) == sp.SPCONV_EINVAL
    n = ctypes.c_int64()
    assert lib.spconv_dense_size(0, 4, 3, 3, ctypes.byref(n)) == sp.SPCONV_EINVAL
    assert lib.spconv_dense_size(8, 4, 3, 3, None) == sp.SPCONV_EINVAL


def test_forward_dense_validates_before_any_gpu_work(sp):
    lib, E, fake = sp._lib, sp.SPCONV_EINVAL, 0x1000

    def call(N=2, C=4, H=8, W=8, K=8, R=3, S=3, pad=1, flags=1, xp=fake, packed=fake, out=fake, epi=None):
        return lib.spconv_forward_dense(xp, N, C, H, W, packed, K, R, S, pad, None, flags,
                                        None if epi is None else ctypes.byref(epi), out, None)

    assert call(xp=None) == E
    assert call(packed=None) == E
    assert call(out=None) == E
    assert call(N=0) == E
    assert call(pad=-1) == E
    assert call(flags=8) == E
    assert call(R=5, S=5, pad=2) == E                  # no 5x5 kernel
    assert call(R=3, S=1) == E
    assert call(H=1, W=1, flags=3) == E                # pool of a 1x1 output
    assert call(W=224, flags=3) == E                   # pool tile wider than 8 blocks
    assert call(epi=sp.spconv_options(-1, 0, None, 0)) == E
    assert call(epi=sp.spconv_options(0, -1, fake, 0)) == E
    info = sp.spconv_plan_info()
    assert lib.spconv_dense_plan(2, 4, 8, 8, 8, 3, 3, 1, 1, None) == E
    assert lib.spconv_dense_plan(2, 4, 8, 8, 8, 3, 3, 1, 1, ctypes.byref(info)) == sp.SPCONV_OK
    assert info.kernel == sp.SPCONV_KERNEL_DENSE and info.workgroups >= 1


def test_dense_plans_cover_the_tile_shapes(sp):
    # 14x14, 256 channels: 4 tiles of 4 rows (two 32-pixel blocks), 4 channel
    # tiles x 2 reduction shares per workgroup, 2048 waves
    p = sp.spconv_dense_plan(32, 256, 14, 14, 256, 3, 3, 1, 1)
    assert (p["tile_rows"], p["pixels_per_lane"], p["threads_per_workgroup"]) == (4, 2, 512)
    # 56x56, 64 channels: 4 rows of 58 padded columns (eight blocks), 2 channel
    # tiles x 2 shares, 1792 waves
    p = sp.spconv_dense_plan(32, 64, 56, 56, 64, 3, 3, 1, 1)
    assert (p["tile_rows"], p["pixels_per_lane"], p["threads_per_workgroup"]) == (4, 8, 256)
    p = sp.spconv_dense_plan(1, 3, 3, 224, 16, 3, 3, 1, 1)
    assert p["pixels_per_lane"] == 8                   # 226 padded columns: eight 32-pixel blocks
    p = sp.spconv_dense_plan(4, 64, 28, 28, 64, 3, 3, 1, 3)
    assert p["tile_rows"] % 2 == 0


def test_select_path(sp):
    sel = sp.spconv_select_path
    full = 256 * 256 * 9
    assert sel(32, 256, 14, 14, 256, 3, 3, 1, 1, int(0.05 * full), 1) == sp.SPCONV_PATH_SPARSE
    assert sel(32, 256, 14, 14, 256, 3, 3, 1, 1, int(0.5 * full), 1) == sp.SPCONV_PATH_DENSE
    assert sel(32, 256, 14, 14, 256, 3, 3, 1, 1, full, 1) == sp.SPCONV_PATH_DENSE
    assert sel(32, 256, 14, 14, 256, 3, 3, 2, 1, full, 1) == sp.SPCONV_PATH_SPARSE   # stride 2: sparse only
    assert sel(32, 64, 14, 14, 64, 5, 5, 1, 2, 64 * 64 * 25, 1) == sp.SPCONV_PATH_SPARSE  # no 5x5 dense kernel
    assert sel(32, 64, 56, 56, 64, 3, 3, 1, 1, 0, 1) == sp.SPCONV_PATH_SPARSE
    # measured break-even: 0.43 at 56x56, 0.245 at 14x14, 0.44 at 28x28 (pooled), 0.67 at 224x224
    assert sel(32, 64, 56, 56, 64, 3, 3, 1, 1, int(0.42 * 64 * 64 * 9), 1) == sp.SPCONV_PATH_SPARSE
    assert sel(32, 64, 56, 56, 64, 3, 3, 1, 1, int(0.44 * 64 * 64 * 9), 1) == sp.SPCONV_PATH_DENSE
    assert sel(32, 256, 14, 14, 256, 3, 3, 1, 1, int(0.23 * full), 1) == sp.SPCONV_PATH_SPARSE
    assert sel(32, 256, 14, 14, 256, 3, 3, 1, 1, int(0.25 * full), 1) == sp.SPCONV_PATH_DENSE
    c128 = 128 * 128 * 9
    assert sel(32, 128, 28, 28, 128, 3, 3, 1, 1, int(0.42 * c128), 3) == sp.SPCONV_PATH_SPARSE
    assert sel(32, 128, 28, 28, 128, 3, 3, 1, 1, int(0.46 * c128), 3) == sp.SPCONV_PATH_DENSE
    c64 = 64 * 64 * 9
    assert sel(32, 64, 224, 224, 64, 3, 3, 1, 1, int(0.65 * c64), 1) == sp.SPCONV_PATH_SPARSE
    assert sel(32, 64, 224, 224, 64, 3, 3, 1, 1, int(0.69 * c64), 1) == sp.SPCONV_PATH_DENSE
    assert sel(32, 64, 224, 224, 64, 3, 3, 1, 1, 64 * 64 * 9, 3) == sp.SPCONV_PATH_SPARSE  # pooled 226-wide rows: no dense plan
    lib, E, out = sp._lib, sp.SPCONV_EINVAL, ctypes.c_int()
    assert lib.spconv_select_path(32, 64, 56, 56, 64, 3, 3, 1, 1, 7280, 1, None) == E
    assert lib.spconv_select_path(32, 64, 56, 56, 64, 3, 3, 1, 1, -1, 1, ctypes.byref(out)) == E
    assert lib.spconv_select_path(32, 64, 56, 56, 64, 3, 3, 1, 1, 64 * 64 * 9 + 1, 1, ctypes.byref(out)) == E
    assert lib.spconv_select_path(32, 64, 56, 56, 64, 3, 3, 0, 1, 7280, 1, ctypes.byref(out)) == E
