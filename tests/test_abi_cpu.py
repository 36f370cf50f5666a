"""Host-side checks of the C-ABI library (no GPU needed).

* libspconv.so loads and exports every function include/spconv.h declares;
* spconv_pack_csr is bit-exact against the oracle's packing (indices and fp32
  bit patterns), including explicit zeros under a mask, -0.0, NaN and empty rows;
* argument validation returns the documented status codes before any GPU work.
"""
import ctypes
import re
from pathlib import Path

import numpy as np
import pytest

import oracle

ROOT = Path(__file__).resolve().parent.parent
HEADER = ROOT / "include" / "spconv.h"


@pytest.fixture(scope="module")
def sp():
    from paper_2005_04091_amd import build
    if not build.LIB_PATH.exists():
        build.build()
    from paper_2005_04091_amd import spconv
    return spconv


def declared_functions():
    text = HEADER.read_text()
    return sorted(set(re.findall(r"^(?:int|const char \*)\s*(spconv_\w+)\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(
        ["spconv_pack_csr", "spconv_pad_input", "spconv_resize_pad_input", "spconv_forward", "spconv_forward_ex",
         "spconv_plan", "spconv_dense_size", "spconv_pack_dense", "spconv_forward_dense", "spconv_dense_plan",
         "spconv_select_path", "spconv_kernel_variants", "spconv_lowered_size", "spconv_pack_lowered",
         "spconv_output_shape", "spconv_strerror"])


def test_library_exports_every_declared_symbol(sp):
    lib = ctypes.CDLL(str(sp.LIB_PATH))
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} not exported"
    assert set(sp.EXPORTED) == set(declared_functions())


def _pack_cases():
    rng = np.random.default_rng(5)
    cases = []
    for i in range(30):
        K, C = int(rng.integers(1, 9)), int(rng.integers(1, 9))
        R, S = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        Hp, Wp = R + int(rng.integers(0, 7)), S + int(rng.integers(0, 7))
        d = [0.0, 0.05, 0.3, 1.0][i % 4]
        w = rng.uniform(-1, 1, (K, C, R, S)).astype(np.float32)
        mask = (rng.random(w.shape) < d).astype(np.uint8)
        w[rng.random(w.shape) < 0.1] = 0.0
        w[rng.random(w.shape) < 0.05] = -0.0
        if i % 3 == 0:
            w[rng.random(w.shape) < 0.05] = np.nan
        if K > 2:
            mask[1] = 0  # an empty row
        cases.append((w, mask, Hp, Wp))
    return cases


@pytest.mark.parametrize("use_mask", [True, False])
def test_pack_matches_oracle_bit_exact(sp, use_mask):
    orc = oracle.get()
    for w, mask, Hp, Wp in _pack_cases():
        m = mask if use_mask else None
        got = sp.spconv_pack_csr(w, m, Hp, Wp)
        rp, ci, off, vals = orc.pack_csr(w, m, Hp, Wp)
        assert np.array_equal(got.rowptr, rp)
        assert np.array_equal(got.colidx, ci)
        assert np.array_equal(got.offset, off)
        assert np.array_equal(got.vals.view(np.uint32), vals.view(np.uint32))


def test_pack_synthetic_configs_bit_exact(sp):
    from paper_2005_04091_amd import synth
    orc = oracle.get()
    for name in ("tiny", "narrow_d0.5"):
        layer = synth.make_layer(name)
        N, C, H, W, K, R, S = layer.shape
        Hp, Wp = H + 2 * layer.pad, W + 2 * layer.pad
        got = sp.spconv_pack_csr(layer.w, layer.mask, Hp, Wp)
        rp, ci, off, vals = orc.pack_csr(layer.w, layer.mask, Hp, Wp)
        assert np.array_equal(got.rowptr, rp) and np.array_equal(got.colidx, ci)
        assert np.array_equal(got.offset, off) and np.array_equal(got.vals.view(np.uint32), vals.view(np.uint32))


def _raw_pack(sp, w, mask, K, C, R, S, Hp, Wp, rowptr, colidx, offset, vals, cap):
    nnz = ctypes.c_int64(-7)
    p = lambda a: None if a is None else a.ctypes.data
    rc = sp._lib.spconv_pack_csr(p(w), p(mask), K, C, R, S, Hp, Wp, p(rowptr), p(colidx), p(offset), p(vals), cap,
                                 ctypes.byref(nnz))
    return rc, nnz.value


def test_pack_count_phase_and_capacity(sp):
    w = np.zeros((2, 1, 3, 3), np.float32)
    w[0, 0, 1, 1] = 2.0
    w[1, 0, 0, 2] = -1.0
    w[1, 0, 2, 0] = 0.5
    rowptr = np.zeros(3, np.int32)
    rc, n = _raw_pack(sp, w, None, 2, 1, 3, 3, 5, 5, rowptr, None, None, None, 0)
    assert rc == sp.SPCONV_OK and n == 3 and rowptr.tolist() == [0, 1, 3]
    ci = np.zeros(2, np.int32)
    off = np.zeros(2, np.int32)
    vals = np.zeros(2, np.float32)
    rc, n = _raw_pack(sp, w, None, 2, 1, 3, 3, 5, 5, rowptr, ci, off, vals, 2)
    assert rc == sp.SPCONV_ECAPACITY and n == 3
    assert ci.tolist() == [0, 0] and vals.tolist() == [0.0, 0.0]


def test_pack_rejects_bad_arguments(sp):
    w = np.ones((2, 2, 3, 3), np.float32)
    rp = np.zeros(3, np.int32)
    ci = np.zeros(36, np.int32)
    off = np.zeros(36, np.int32)
    v = np.zeros(36, np.float32)
    E = sp.SPCONV_EINVAL
    assert _raw_pack(sp, None, None, 2, 2, 3, 3, 5, 5, rp, ci, off, v, 36)[0] == E
    assert _raw_pack(sp, w, None, 0, 2, 3, 3, 5, 5, rp, ci, off, v, 36)[0] == E
    assert _raw_pack(sp, w, None, 2, 2, 3, 3, 2, 5, rp, ci, off, v, 36)[0] == E  # Hp < R
    assert _raw_pack(sp, w, None, 2, 2, 3, 3, 5, 2, rp, ci, off, v, 36)[0] == E  # Wp < S
    assert _raw_pack(sp, w, None, 2, 2, 3, 3, 5, 5, rp, ci, None, v, 36)[0] == E  # partial outputs
    assert _raw_pack(sp, w, None, 2, 2, 3, 3, 5, 5, None, ci, off, v, 36)[0] == E  # fill without rowptr
    assert _raw_pack(sp, w, None, 2, 2, 3, 3, 5, 5, rp, ci, off, v, -1)[0] == E
    # offsets that would not fit int32
    assert _raw_pack(sp, w, None, 2, 2, 3, 3, 50000, 50000, rp, ci, off, v, 36)[0] == E


def test_output_shape(sp):
    assert sp.spconv_output_shape(56, 56, 3, 3, 1, 1, sp.SPCONV_RELU) == (56, 56)
    assert sp.spconv_output_shape(28, 28, 3, 3, 1, 1, sp.SPCONV_RELU | sp.SPCONV_MAXPOOL2X2) == (14, 14)
    assert sp.spconv_output_shape(7, 9, 3, 3, 2, 1, 0) == (4, 5)
    assert sp.spconv_output_shape(5, 5, 3, 3, 1, 1, sp.SPCONV_MAXPOOL2X2) == (2, 2)  # odd: floor
    assert sp.spconv_output_shape(56, 56, 3, 3, 1, 1, sp.SPCONV_RELU | sp.SPCONV_UNPADDED_INPUT) == (56, 56)
    for bad in [(0, 5, 3, 3, 1, 1, 0), (5, 5, 3, 3, 0, 1, 0), (5, 5, 3, 3, 1, -1, 0), (5, 5, 3, 3, 1, 1, 8),
                (2, 2, 3, 3, 1, 0, 0), (3, 3, 3, 3, 1, 0, sp.SPCONV_MAXPOOL2X2)]:
        with pytest.raises(sp.SpconvError) as e:
            sp.spconv_output_shape(*bad)
        assert e.value.code == sp.SPCONV_EINVAL


def test_strerror(sp):
    for code in (0, -1, -2, -3, 99):
        assert isinstance(sp.spconv_strerror(code), str) and sp.spconv_strerror(code)
    assert sp.spconv_strerror(-1) != sp.spconv_strerror(-2)


def test_forward_and_pad_validate_before_any_gpu_work(sp):
    """Every call below is invalid and must return SPCONV_EINVAL from the host
    checks; fake (never dereferenced) addresses stand in for device buffers."""
    lib = sp._lib
    E = sp.SPCONV_EINVAL
    fake = 0x1000
    csr = sp.spconv_csr(4, 3, 3, 3, 10, 12, 5, fake, fake, fake, fake)
    ok = dict(xp=fake, N=2, C=3, H=8, W=10, K=4, R=3, S=3, stride=1, pad=1, bias=None, flags=1, out=fake)

    def fwd(**kw):
        a = dict(ok)
        a.update(kw)
        c = kw.get("csr", csr)
        return lib.spconv_forward(a["xp"], a["N"], a["C"], a["H"], a["W"], ctypes.byref(c), a["K"], a["R"], a["S"],
                                  a["stride"], a["pad"], a["bias"], a["flags"], a["out"], None)

    assert fwd(xp=None) == E
    assert fwd(out=None) == E
    assert lib.spconv_forward(fake, 2, 3, 8, 10, None, 4, 3, 3, 1, 1, None, 1, fake, None) == E
    assert fwd(N=0) == E
    assert fwd(stride=0) == E
    assert fwd(pad=-1) == E
    assert fwd(flags=8) == E
    assert fwd(stride=2, flags=1 | sp.SPCONV_UNPADDED_INPUT) == E  # unpadded input: stride-1 plans only
    assert fwd(K=5) == E            # csr->K mismatch
    assert fwd(C=4) == E            # csr->C mismatch
    assert fwd(H=9) == E            # csr->Hp != H + 2 pad
    assert fwd(pad=2) == E          # csr->Hp/Wp mismatch
    bad_nnz = sp.spconv_csr(4, 3, 3, 3, 10, 12, -1, fake, fake, fake, fake)
    assert fwd(csr=bad_nnz) == E
    null_rows = sp.spconv_csr(4, 3, 3, 3, 10, 12, 5, None, fake, fake, fake)
    assert fwd(csr=null_rows) == E
    tiny = sp.spconv_csr(4, 3, 3, 3, 3, 3, 5, fake, fake, fake, fake)
    assert fwd(csr=tiny, H=3, W=3, pad=0, flags=sp.SPCONV_MAXPOOL2X2) == E  # 1x1 output cannot be pooled
    # epilogue options are checked on the host as well
    def fwd_ex(out_pad=0, residual_pad=0, residual=None, max_row_nnz=0, **kw):
        a = dict(ok)
        a.update(kw)
        opt = sp.spconv_options(out_pad, residual_pad, residual, max_row_nnz)
        return lib.spconv_forward_ex(a["xp"], a["N"], a["C"], a["H"], a["W"], ctypes.byref(csr), a["K"], a["R"],
                                     a["S"], a["stride"], a["pad"], a["bias"], a["flags"], ctypes.byref(opt),
                                     a["out"], None)

    for bad_hint in (-1, 6):        # the largest row cannot have more entries than the filter
        assert fwd_ex(max_row_nnz=bad_hint) == E

    assert fwd_ex(out_pad=-1) == E
    assert fwd_ex(residual=fake, residual_pad=-1) == E
    assert fwd_ex(out_pad=1 << 16) == E            # padded output plane of 2^31 elements or more
    assert fwd_ex(residual=fake, residual_pad=1 << 16) == E
    assert fwd_ex(out=None, out_pad=1) == E
    assert fwd_ex(N=0, out_pad=1) == E
    assert lib.spconv_pad_input(None, 1, 1, 4, 4, 1, fake, None) == E
    assert lib.spconv_pad_input(fake, 1, 1, 0, 4, 1, fake, None) == E
    assert lib.spconv_pad_input(fake, 1, 1, 4, 4, -1, fake, None) == E
    assert lib.spconv_pad_input(fake, 1, 1, 4, 4, 1, None, None) == E
    assert lib.spconv_pad_input(fake, 1, 1, 1, (1 << 31) - 4000, 0, fake, None) == E  # plane above 2^31 - 4096
    rz = lib.spconv_resize_pad_input
    assert rz(None, 1, 1, 4, 4, 2, 2, 1, fake, None) == E
    assert rz(fake, 1, 1, 4, 4, 2, 2, 1, None, None) == E
    assert rz(fake, 0, 1, 4, 4, 2, 2, 1, fake, None) == E
    assert rz(fake, 1, 1, 0, 4, 2, 2, 1, fake, None) == E
    assert rz(fake, 1, 1, 4, 4, 2, 0, 1, fake, None) == E
    assert rz(fake, 1, 1, 4, 4, 2, 2, -1, fake, None) == E
    assert rz(fake, 1, 1, 16385, 4, 2, 2, 1, fake, None) == E      # a side above 16384
    assert rz(fake, 1, 1, 4, 4, 2, 16385, 0, fake, None) == E
    assert rz(fake, 1, 1, 4, 4, 2, 2, 1 << 15, fake, None) == E    # padded plane of 2^31 elements or more
    assert rz(fake, 1 << 20, 1 << 10, 4, 4, 32, 32, 0, fake, None) == E  # 2^40 output elements
    assert rz(fake, 1 << 20, 1 << 10, 32, 32, 2, 2, 0, fake, None) == E  # 2^40 input elements


def test_plan_reports_the_launch_without_a_gpu(sp):
    """spconv_plan runs the forward call's host checks and planner only; fake
    (never dereferenced) addresses stand in for the CSR arrays."""
    lib = sp._lib
    fake = 0x1000

    def plan(N, C, H, W, K, R=3, S=3, stride=1, pad=1, flags=sp.SPCONV_RELU, nnz=None, max_row=0):
        nnz = int(0.2 * K * C * R * S) if nnz is None else nnz
        csr = sp.spconv_csr(K, C, R, S, H + 2 * pad, W + 2 * pad, nnz, fake, fake, fake, fake)
        opt = sp.spconv_options(0, 0, None, max_row)
        info = sp.spconv_plan_info()
        rc = lib.spconv_plan(N, C, H, W, ctypes.byref(csr), K, R, S, stride, pad, flags, ctypes.byref(opt),
                             ctypes.byref(info))
        return rc, info

    rc, p = plan(32, 64, 56, 56, 64)                      # ResNet-style layer
    assert rc == sp.SPCONV_OK
    assert p.kernel == sp.SPCONV_KERNEL_STRIDE1 and p.threads_per_workgroup == 1024
    # the grid covers every (image group, spatial tile, channel tile) exactly once
    kt = 16 * p.channels_per_wave
    assert p.workgroups == -(-32 // p.images_per_group) * p.tiles_per_image * -(-64 // kt)
    assert p.tile_rows * p.tiles_per_image >= 56 and p.tile_rows * (p.tiles_per_image - 1) < 56
    assert p.channels_per_chunk * p.chunks >= 64 and p.channels_per_chunk * (p.chunks - 1) < 64
    assert 0 < p.lds_bytes <= 160 * 1024
    # a filter with a dense channel makes the planner pair channels per wave
    rc, flat = plan(32, 256, 14, 14, 256, nnz=117965, max_row=117965 // 256)
    rc2, skewed = plan(32, 256, 14, 14, 256, nnz=117965, max_row=3 * 117965 // 256)
    assert rc == rc2 == sp.SPCONV_OK and skewed.channels_per_wave >= 2
    rc, p = plan(2, 5, 9, 8, 7, stride=2)                   # strided layers take the any-stride kernel
    assert rc == sp.SPCONV_OK and p.kernel == sp.SPCONV_KERNEL_GENERIC
    assert plan(2, 5, 9, 8, 7, max_row=10 ** 9)[0] == sp.SPCONV_EINVAL  # hint above nnz
    assert plan(2, 5, 9, 8, 7, flags=8)[0] == sp.SPCONV_EINVAL
    csr = sp.spconv_csr(7, 5, 3, 3, 11, 10, 60, fake, fake, fake, fake)
    assert lib.spconv_plan(2, 5, 9, 8, ctypes.byref(csr), 7, 3, 3, 1, 1, 1, None, None) == sp.SPCONV_EINVAL
    # options are optional: NULL plans like a zero struct
    info = sp.spconv_plan_info()
    assert lib.spconv_plan(2, 5, 9, 8, ctypes.byref(csr), 7, 3, 3, 1, 1, 1, None, ctypes.byref(info)) == sp.SPCONV_OK
    opt = sp.spconv_options(-1, 0, None, 0)
    assert lib.spconv_plan(2, 5, 9, 8, ctypes.byref(csr), 7, 3, 3, 1, 1, 1, ctypes.byref(opt),
                           ctypes.byref(info)) == sp.SPCONV_EINVAL


def test_plans_fit_the_lds_over_a_sweep_of_shapes(sp):
    """Every stride-1 plan fits one CU's 160 KiB of LDS (chunk buffers rounded to
    64 floats, the slack after them, the pooled staging area), and every dense
    plan its 64 KiB, over widths, heights, channel counts, batch sizes and
    pooling; the grid covers each (image group, tile, channel tile) once."""
    lib = sp._lib
    fake = 0x1000
    seen = seen_dense = 0
    for N in (1, 3, 32):
        for C in (1, 3, 16, 64, 130, 512):
            for H, W in ((2, 2), (7, 9), (14, 14), (28, 28), (56, 56), (61, 70), (224, 224), (5, 600)):
                for pool in (False, True):
                    flags = sp.SPCONV_RELU | (sp.SPCONV_MAXPOOL2X2 if pool else 0)
                    K = 64
                    nnz = max(1, int(0.2 * K * C * 9))
                    csr = sp.spconv_csr(K, C, 3, 3, H + 2, W + 2, nnz, fake, fake, fake, fake)
                    info = sp.spconv_plan_info()
                    rc = lib.spconv_plan(N, C, H, W, ctypes.byref(csr), K, 3, 3, 1, 1, flags, None,
                                         ctypes.byref(info))
                    if rc != sp.SPCONV_OK:
                        continue
                    seen += 1
                    assert 0 < info.lds_bytes <= 160 * 1024, (N, C, H, W, pool, info.lds_bytes)
                    if info.kernel == sp.SPCONV_KERNEL_STRIDE1:
                        kt = 16 * info.channels_per_wave
                        assert info.workgroups == -(-N // info.images_per_group) * info.tiles_per_image * -(-K // kt)
                        assert info.channels_per_chunk * info.chunks >= C
                    dinfo = sp.spconv_plan_info()
                    if lib.spconv_dense_plan(N, C, H, W, K, 3, 3, 1, flags, ctypes.byref(dinfo)) == sp.SPCONV_OK:
                        seen_dense += 1
                        assert 0 < dinfo.lds_bytes <= 64 * 1024, (N, C, H, W, pool, dinfo.lds_bytes)
    assert seen > 200 and seen_dense > 100
