"""Pins that tie the CPU oracle to facts outside itself.

Each pin takes an oracle object (``oracle.Oracle``: the real build, or a planted
mutant built by the mutant test) and raises AssertionError when the oracle
disagrees with:

* a library routine for the special case the method reduces to
  (``torch.nn.functional.conv2d`` / ``max_pool2d`` in float64, ``scipy.sparse``'s
  CSR of the flattened filter, ``numpy.ravel_multi_index`` for padded offsets);
* closed forms (all-ones filter, identity filter, single-tap shifts, zero density,
  power-of-two scaling);
* worked examples under ``tests/golden/`` derived by hand from the paper's
  definitions (the dense convolution of the DSL section, the CSR flattening of
  "Sparse Convolution with CSR").
"""
from __future__ import annotations

import json
from pathlib import Path

import numpy as np
import scipy.sparse
import torch
import torch.nn.functional as F

GOLDEN = Path(__file__).resolve().parent / "golden"


def _rng(seed):
    return np.random.default_rng(seed)


def _torch_block(x, w_eff, bias, stride, pad, relu, pool):
    """Library witness: conv2d (cross-correlation) -> bias -> ReLU -> 2x2 max-pool, float64."""
    X = torch.from_numpy(np.asarray(x, np.float64))
    Wt = torch.from_numpy(np.asarray(w_eff, np.float64))
    B = None if bias is None else torch.from_numpy(np.asarray(bias, np.float64))
    y = F.conv2d(X, Wt, bias=B, stride=stride, padding=pad)
    if relu:
        y = torch.relu(y)
    if pool:
        y = F.max_pool2d(y, kernel_size=2, stride=2)
    return y.numpy()


def _random_case(rng, allow_masked_values=True):
    N = int(rng.integers(1, 3))
    C = int(rng.integers(1, 6))
    K = int(rng.integers(1, 6))
    R = int(rng.integers(1, 4))
    S = int(rng.integers(1, 4))
    stride = int(rng.integers(1, 3))
    pad = int(rng.integers(0, 3))
    H = int(rng.integers(max(R, 2), 10))
    W = int(rng.integers(max(S, 2), 10))
    if H + 2 * pad == R:
        H += 1
    if W + 2 * pad == S:
        W += 1
    x = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    w = rng.uniform(-1, 1, (K, C, R, S)).astype(np.float32)
    mask = (rng.random((K, C, R, S)) < 0.5).astype(np.uint8)
    if not allow_masked_values:
        w = np.where(mask != 0, w, 0).astype(np.float32)
    bias = rng.uniform(-0.5, 0.5, K).astype(np.float32) if rng.random() < 0.7 else None
    return x, w, mask, bias, stride, pad


def pin_library_conv(orc):
    """Oracle == float64 conv2d -> ReLU -> max_pool2d on random small shapes,
    with the mask applied (masked-off positions hold nonzero values that must be
    ignored), odd/even sizes, R != S, stride 1/2, pad 0..2."""
    rng = _rng(11)
    for _ in range(40):
        x, w, mask, bias, stride, pad = _random_case(rng)
        w_eff = w * mask
        for relu, pool in ((False, False), (True, False), (True, True), (False, True)):
            Ho = (x.shape[2] + 2 * pad - w.shape[2]) // stride + 1
            Wo = (x.shape[3] + 2 * pad - w.shape[3]) // stride + 1
            if pool and (Ho < 2 or Wo < 2):
                continue
            got, ab = orc.conv(x, w, mask, bias, stride, pad, relu, pool)
            ref = _torch_block(x, w_eff, bias, stride, pad, relu, pool)
            assert got.shape == ref.shape, (got.shape, ref.shape)
            scale = ab + (0 if bias is None else np.abs(bias).max()) + 1e-30
            assert np.all(np.abs(got - ref) <= 1e-12 * scale), "conv differs from conv2d"


def pin_library_absacc(orc):
    """absacc == conv2d(|x|, |w*mask|) (max-pooled when pooling): the sum of |w*x|."""
    rng = _rng(12)
    for _ in range(20):
        x, w, mask, bias, stride, pad = _random_case(rng)
        for pool in (False, True):
            Ho = (x.shape[2] + 2 * pad - w.shape[2]) // stride + 1
            Wo = (x.shape[3] + 2 * pad - w.shape[3]) // stride + 1
            if pool and (Ho < 2 or Wo < 2):
                continue
            _, ab = orc.conv(x, w, mask, bias, stride, pad, True, pool)
            ref = _torch_block(np.abs(x), np.abs(w * mask), None, stride, pad, False, pool)
            assert np.all(np.abs(ab - ref) <= 1e-12 * (ref + 1e-30)), "absacc differs"


def pin_hand_example(orc):
    """The hand-worked 3x3 example in tests/golden/hand_conv_3x3.json."""
    g = json.loads((GOLDEN / "hand_conv_3x3.json").read_text())
    x = np.array(g["x"], np.float32)[None, None]
    w = np.array(g["w"], np.float32)[None, None]
    pad = g["pad"]
    out, ab = orc.conv(x, w, None, None, 1, pad, False, False)
    assert np.array_equal(out[0, 0], np.array(g["pre_stride1"], np.float64)), out[0, 0]
    assert np.array_equal(ab[0, 0], np.array(g["absacc_stride1"], np.float64)), ab[0, 0]
    b = np.array([g["bias"]], np.float32)
    out, _ = orc.conv(x, w, None, b, 1, pad, True, False)
    assert np.array_equal(out[0, 0], np.array(g["relu_bias_stride1"], np.float64)), out[0, 0]
    out, ab = orc.conv(x, w, None, b, 1, pad, True, True)
    assert np.array_equal(out[0, 0], np.array(g["relu_bias_pool"], np.float64)), out[0, 0]
    assert np.array_equal(ab[0, 0], np.array(g["absacc_pool"], np.float64)), ab[0, 0]
    out, _ = orc.conv(x, w, None, None, 2, pad, False, False)
    assert np.array_equal(out[0, 0], np.array(g["pre_stride2"], np.float64)), out[0, 0]


def pin_identity_filter(orc):
    """C == K, one 1.0 per row at (c=k, centre tap), pad = R//2, stride 1: the
    output reproduces the (non-negative) input bit for bit, and with pooling it is
    the 2x2 block max of the input."""
    rng = _rng(13)
    for (R, S, H, W) in ((3, 3, 7, 9), (1, 1, 4, 6), (5, 5, 8, 8), (3, 3, 6, 10)):
        C = 4
        x = rng.random((2, C, H, W), dtype=np.float32)
        w = np.zeros((C, C, R, S), np.float32)
        for k in range(C):
            w[k, k, R // 2, S // 2] = 1.0
        out, _ = orc.conv(x, w, None, None, 1, R // 2, True, False)
        assert np.array_equal(out, x.astype(np.float64)), "identity filter changed the input"
        out, _ = orc.conv(x, w, None, None, 1, R // 2, True, True)
        ref = x[:, :, : H // 2 * 2, : W // 2 * 2].reshape(2, C, H // 2, 2, W // 2, 2).max(axis=(3, 5))
        assert np.array_equal(out, ref.astype(np.float64)), "identity filter + pool"


def pin_all_ones(orc):
    """All-ones 3x3 filter and input, pad 1: output = b + C * (#taps inside the
    image): 9C inside, 6C on edges, 4C at corners."""
    N, C, K, H, W = 1, 5, 2, 6, 7
    x = np.ones((N, C, H, W), np.float32)
    w = np.ones((K, C, 3, 3), np.float32)
    b = np.array([0.25, -0.5], np.float32)
    out, _ = orc.conv(x, w, None, b, 1, 1, False, False)
    rows = np.array([2 if y in (0, H - 1) else 3 for y in range(H)], np.float64)
    cols = np.array([2 if q in (0, W - 1) else 3 for q in range(W)], np.float64)
    taps = rows[:, None] * cols[None, :]
    for k in range(K):
        assert np.array_equal(out[0, k], b[k] + C * taps), "all-ones closed form"
    assert out[0, 0, 0, 0] == b[0] + 4 * C and out[0, 0, 0, 3] == b[0] + 6 * C and out[0, 0, 3, 3] == b[0] + 9 * C


def pin_single_tap_shift(orc):
    """Filter row k has one 1.0 at (c_k, r_k, s_k): its output is channel c_k of the
    input shifted by (r_k - pad, s_k - pad) (and strided), zero where it reads the
    padding."""
    rng = _rng(14)
    for stride in (1, 2):
        N, C, H, W, R, S, pad = 2, 3, 7, 8, 3, 4, 2
        K = 6
        x = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
        w = np.zeros((K, C, R, S), np.float32)
        taps = [(int(rng.integers(C)), int(rng.integers(R)), int(rng.integers(S))) for _ in range(K)]
        for k, (c, r, s) in enumerate(taps):
            w[k, c, r, s] = 1.0
        out, _ = orc.conv(x, w, None, None, stride, pad, False, False)
        Ho = (H + 2 * pad - R) // stride + 1
        Wo = (W + 2 * pad - S) // stride + 1
        for k, (c, r, s) in enumerate(taps):
            for y in range(Ho):
                for q in range(Wo):
                    iy, ix = y * stride + r - pad, q * stride + s - pad
                    v = x[:, c, iy, ix] if (0 <= iy < H and 0 <= ix < W) else np.zeros(N, np.float32)
                    assert np.array_equal(out[:, k, y, q], v.astype(np.float64)), (k, y, q)


def pin_zero_density(orc):
    """No entries: output = act(bias) everywhere (and 0 without bias)."""
    x = _rng(15).random((2, 3, 5, 6), dtype=np.float32)
    w = np.ones((4, 3, 3, 3), np.float32)
    mask = np.zeros(w.shape, np.uint8)
    b = np.array([-0.3, 0.0, 0.2, 1.5], np.float32)
    out, ab = orc.conv(x, w, mask, b, 1, 1, True, False)
    for k in range(4):
        assert np.all(out[:, k] == max(float(b[k]), 0.0))
    assert np.all(ab == 0)
    out, _ = orc.conv(x, w, mask, b, 1, 1, False, True)
    for k in range(4):
        assert np.all(out[:, k] == float(b[k]))


def pin_power_of_two_scaling(orc):
    """Scaling weights and bias by 2**e scales the pre-activation exactly."""
    rng = _rng(16)
    x, w, mask, bias, stride, pad = _random_case(rng)
    bias = rng.uniform(-1, 1, w.shape[0]).astype(np.float32)
    base, _ = orc.conv(x, w, mask, bias, stride, pad, False, False)
    for e in (-3, 5):
        sc, _ = orc.conv(x, w * np.float32(2.0 ** e), mask, bias * np.float32(2.0 ** e), stride, pad, False, False)
        assert np.array_equal(sc, base * 2.0 ** e), "power-of-two scaling"


def pin_pool_invariants(orc):
    """Pooled output = max of the four un-pooled outputs of its window (floor at
    odd sizes); the max is one of them; with ReLU it is >= 0."""
    rng = _rng(17)
    for _ in range(10):
        x, w, mask, bias, stride, pad = _random_case(rng)
        Ho = (x.shape[2] + 2 * pad - w.shape[2]) // stride + 1
        Wo = (x.shape[3] + 2 * pad - w.shape[3]) // stride + 1
        if Ho < 2 or Wo < 2:
            continue
        for relu in (False, True):
            full, _ = orc.conv(x, w, mask, bias, stride, pad, relu, False)
            pooled, _ = orc.conv(x, w, mask, bias, stride, pad, relu, True)
            Hq, Wq = Ho // 2, Wo // 2
            win = full[:, :, : 2 * Hq, : 2 * Wq].reshape(full.shape[0], full.shape[1], Hq, 2, Wq, 2)
            assert np.array_equal(pooled, win.max(axis=(3, 5))), "pool != max of window"
            if relu:
                assert np.all(pooled >= 0)


def pin_csr_library(orc):
    """rowptr/colidx/vals == scipy.sparse CSR of the (K, C*R*S) flattened filter:
    with a mask, the stored positions are the mask's (explicit 0.0 values stay);
    without one, the nonzero values (-0.0 dropped, NaN kept)."""
    rng = _rng(18)
    for _ in range(25):
        K, C, R, S = (int(v) for v in rng.integers(1, 6, 4))
        Hp, Wp = R + int(rng.integers(0, 4)), S + int(rng.integers(0, 4))
        w = rng.uniform(-1, 1, (K, C, R, S)).astype(np.float32)
        w[rng.random(w.shape) < 0.2] = 0.0
        w[rng.random(w.shape) < 0.1] = -0.0
        mask = (rng.random(w.shape) < 0.5).astype(np.uint8)
        mask[mask != 0] = rng.integers(1, 256, int(mask.sum()), dtype=np.uint8)
        flat = w.reshape(K, -1)
        rows, cols = np.nonzero(mask.reshape(K, -1))
        ref_m = scipy.sparse.coo_matrix((flat[rows, cols], (rows, cols)), shape=flat.shape).tocsr()
        ref_m.sort_indices()
        rp, ci, off, vals = orc.pack_csr(w, mask, Hp, Wp)
        assert np.array_equal(rp, ref_m.indptr.astype(np.int32)), "rowptr (masked)"
        assert np.array_equal(ci, ref_m.indices.astype(np.int32)), "colidx (masked)"
        assert np.array_equal(vals.view(np.uint32), ref_m.data.astype(np.float32).view(np.uint32)), "vals (masked)"
        wn = w.copy()
        wn[0, 0, 0, 0] = np.nan
        ref_n = scipy.sparse.csr_matrix(wn.reshape(K, -1))
        ref_n.sort_indices()
        rp, ci, off, vals = orc.pack_csr(wn, None, Hp, Wp)
        assert np.array_equal(rp, ref_n.indptr.astype(np.int32)), "rowptr (values)"
        assert np.array_equal(ci, ref_n.indices.astype(np.int32)), "colidx (values)"
        assert np.array_equal(vals.view(np.uint32), ref_n.data.astype(np.float32).view(np.uint32)), "vals (values)"


def pin_csr_offsets(orc):
    """Each offset is the flat index of tap (c, r, s) in a C x Hp x Wp padded image
    (numpy.ravel_multi_index), with (c, r, s) decoded from colidx by divmod."""
    rng = _rng(19)
    for _ in range(25):
        K, C, R, S = (int(v) for v in rng.integers(1, 6, 4))
        Hp, Wp = R + int(rng.integers(0, 5)), S + int(rng.integers(0, 5))
        w = rng.uniform(-1, 1, (K, C, R, S)).astype(np.float32)
        mask = (rng.random(w.shape) < 0.4).astype(np.uint8)
        rp, ci, off, vals = orc.pack_csr(w, mask, Hp, Wp)
        c, rs = np.divmod(ci, R * S)
        r, s = np.divmod(rs, S)
        ref = np.ravel_multi_index((c, r, s), (C, Hp, Wp)).astype(np.int32)
        assert np.array_equal(off, ref), "offset formula"
        # Round trip: scattering the entries back gives w * mask bit for bit.
        dense = np.zeros((K, C * R * S), np.float32)
        rows = np.repeat(np.arange(K), np.diff(rp))
        dense[rows, ci] = vals
        ref_dense = np.where(mask.reshape(K, -1) != 0, w.reshape(K, -1), np.float32(0.0)).astype(np.float32)
        assert np.array_equal(dense.view(np.uint32), ref_dense.view(np.uint32)), "round trip"
        assert np.all(np.diff(rp) >= 0) and rp[0] == 0 and rp[-1] == ci.size
        for k in range(K):
            assert np.all(np.diff(ci[rp[k]:rp[k + 1]]) > 0), "colidx not increasing within a row"


def pin_csr_golden(orc):
    """The hand-worked CSR example in tests/golden/csr_tiny.json."""
    g = json.loads((GOLDEN / "csr_tiny.json").read_text())
    w = np.array(g["w"], np.float32)
    rp, ci, off, vals = orc.pack_csr(w, None, g["Hp"], g["Wp"])
    assert rp.tolist() == g["rowptr"] and ci.tolist() == g["colidx"] and off.tolist() == g["offset"]
    assert vals.tolist() == g["vals"]


def pin_library_residual(orc):
    """With a residual (the shortcut of a ResNet basic block): oracle ==
    float64 conv2d + bias + residual -> ReLU -> max_pool2d, the residual on the
    convolution's own grid, added before the activation and the pool; and its
    sum of |w*x| grows by |residual| exactly."""
    rng = _rng(31)
    for _ in range(25):
        x, w, mask, bias, stride, pad = _random_case(rng)
        w_eff = w * mask
        N, K = x.shape[0], w.shape[0]
        Ho = (x.shape[2] + 2 * pad - w.shape[2]) // stride + 1
        Wo = (x.shape[3] + 2 * pad - w.shape[3]) // stride + 1
        res = rng.uniform(-2, 2, (N, K, Ho, Wo)).astype(np.float32)
        for relu, pool in ((False, False), (True, False), (True, True)):
            if pool and (Ho < 2 or Wo < 2):
                continue
            got, ab = orc.conv(x, w, mask, bias, stride, pad, relu, pool, residual=res)
            y = _torch_block(x, w_eff, bias, stride, pad, False, False) + res.astype(np.float64)
            if relu:
                y = np.maximum(y, 0.0)
            if pool:
                y = F.max_pool2d(torch.from_numpy(y), kernel_size=2, stride=2).numpy()
            assert got.shape == y.shape, (got.shape, y.shape)
            assert np.allclose(got, y, rtol=1e-12, atol=1e-12), float(np.abs(got - y).max())
        _, ab0 = orc.conv(x, w, mask, bias, stride, pad, False, False)
        _, ab1 = orc.conv(x, w, mask, bias, stride, pad, False, False, residual=res)
        assert np.allclose(ab1 - ab0, np.abs(res.astype(np.float64)), rtol=0, atol=1e-12)


def pin_residual_closed_forms(orc):
    """Zero filter: out = relu(b + res) exactly. Identity filter (one 1.0 at
    (c = k, centre tap), pad 1): out = relu(x + res), and pooled its 2x2 max."""
    rng = _rng(32)
    N, C, H, W = 2, 3, 6, 8
    x = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    res = rng.uniform(-1, 1, (N, C, H, W)).astype(np.float32)
    b = rng.uniform(-0.5, 0.5, C).astype(np.float32)
    w0 = np.zeros((C, C, 3, 3), np.float32)
    got, _ = orc.conv(x, w0, None, b, 1, 1, True, False, residual=res)
    want = np.maximum(b[None, :, None, None].astype(np.float64) + res, 0.0)
    assert np.array_equal(got, want)
    wi = np.zeros((C, C, 3, 3), np.float32)
    for k in range(C):
        wi[k, k, 1, 1] = 1.0
    got, _ = orc.conv(x, wi, None, None, 1, 1, True, False, residual=res)
    want = np.maximum(x.astype(np.float64) + res.astype(np.float64), 0.0)
    assert np.array_equal(got, want)
    gp, _ = orc.conv(x, wi, None, None, 1, 1, True, True, residual=res)
    wp = want.reshape(N, C, H // 2, 2, W // 2, 2).max(axis=(3, 5))
    assert np.array_equal(gp, wp)


def _torch_resize(x, H, W):
    X = torch.from_numpy(np.asarray(x, np.float64))
    return F.interpolate(X, size=(H, W), mode="bilinear", align_corners=False).numpy()


def pin_resize_library(orc):
    """Bilinear resize (half-pixel centres) == float64
    torch.nn.functional.interpolate(mode="bilinear", align_corners=False) on
    random shapes: up, down, non-integer ratios, H != W, one-pixel planes; and
    its sum of |w*v| == the same interpolation of |x| (the weights are >= 0)."""
    rng = _rng(41)
    for _ in range(40):
        N, C = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        Hin, Win = int(rng.integers(1, 12)), int(rng.integers(1, 12))
        H, W = int(rng.integers(1, 25)), int(rng.integers(1, 25))
        x = rng.uniform(-1, 1, (N, C, Hin, Win)).astype(np.float32)
        got, ab = orc.resize(x, H, W)
        ref = _torch_resize(x, H, W)
        assert np.allclose(got, ref, rtol=0, atol=1e-12), float(np.abs(got - ref).max())
        assert np.allclose(ab, _torch_resize(np.abs(x), H, W), rtol=0, atol=1e-12)


def pin_resize_closed_forms(orc):
    """Same size: an exact copy. Exact factor-2 downsampling: the mean of each
    2x2 block. A constant plane stays constant at any size (the four weights
    sum to one up to double rounding)."""
    rng = _rng(42)
    x = rng.uniform(-1, 1, (2, 3, 6, 10)).astype(np.float32)
    got, _ = orc.resize(x, 6, 10)
    assert np.array_equal(got, x.astype(np.float64))
    got, _ = orc.resize(x, 3, 5)
    ref = x.astype(np.float64).reshape(2, 3, 3, 2, 5, 2).mean(axis=(3, 5))
    assert np.allclose(got, ref, rtol=0, atol=1e-15)
    c = np.full((1, 2, 5, 7), 0.75, np.float32)
    for H, W in ((1, 1), (9, 3), (10, 14), (4, 4)):
        got, _ = orc.resize(c, H, W)
        assert np.allclose(got, 0.75, rtol=0, atol=1e-15)


ALL_PINS = [
    pin_library_conv,
    pin_library_absacc,
    pin_hand_example,
    pin_identity_filter,
    pin_all_ones,
    pin_single_tap_shift,
    pin_zero_density,
    pin_power_of_two_scaling,
    pin_pool_invariants,
    pin_csr_library,
    pin_csr_offsets,
    pin_csr_golden,
    pin_library_residual,
    pin_residual_closed_forms,
    pin_resize_library,
    pin_resize_closed_forms,
]
