"""Host-side checks of the lowered entry stream (no GPU needed).

``spconv_pack_lowered`` is compared word for word with an independent numpy
construction of the layout include/spconv.h documents (headers per (tile, wave,
slot, chunk), entries re-based to the plan's staged tile and split by tap
parity), given the packer's assignment of rows to (wave, slot), which is
checked to cover each channel tile's rows once and to balance the chunks' work
no worse than the snake deal by entry count it starts from, over layers whose
plans cover one, two and four rows per wave, one and several chunks, several
images per tile, pooling and the unpadded-input tile geometry; its errors and
the forward call's checks of a stream are exercised with never-dereferenced
addresses.
"""
import ctypes

import numpy as np
import pytest

from paper_2005_04091_amd import synth


@pytest.fixture(scope="module")
def sp():
    from paper_2005_04091_amd import spconv
    return spconv


def snake_slots(host, K, kt, rpw):
    """The snake deal by entry count that the packer starts from: {(wave, slot): row}."""
    rp = host.rowptr
    kt_rows = 16 * rpw
    k0 = kt * kt_rows
    nz = [int(rp[k0 + j + 1] - rp[k0 + j]) if k0 + j < K else -1 for j in range(kt_rows)]
    order = sorted(range(kt_rows), key=lambda j: (-nz[j], j)) if rpw > 1 else list(range(kt_rows))
    slot = {}
    for rank, j in enumerate(order):
        i, w = divmod(rank, 16)
        slot[(15 - w if i % 2 else w, i)] = k0 + j
    return slot


AGE_SHARE = np.array([120, 107, 93, 80], np.int64)  # issue share of wave 4*g + s, by age group g


def chunk_costs(host, plan, K, C, R, S, slots):
    """Sum over chunks of the busiest SIMD's cost, max(SIMD entries, each of
    its waves' entries scaled by the wave's age share), for one channel tile's
    {(wave, slot): row}."""
    rp, ci = host.rowptr, host.colidx
    cc, nch = plan["channels_per_chunk"], plan["chunks"]
    load = np.zeros((16, nch), np.int64)
    for (w, i), k in slots.items():
        if k < K:
            for j in range(rp[k], rp[k + 1]):
                load[w, (int(ci[j]) // (R * S)) // cc] += 1
    per_simd = load.reshape(4, 4, nch)   # wave w = 4 * g + s runs on SIMD s
    scaled = per_simd * AGE_SHARE.sum() * 1000 // AGE_SHARE[:, None, None]
    return int(np.maximum(per_simd.sum(axis=0) * 1000, scaled.max(axis=0)).max(axis=0).sum())


def packed_slots(got, plan, K, kt):
    """{(wave, slot): row} of one channel tile, read from the stream's headers (chunk 0)."""
    rpw, nch = plan["channels_per_wave"], plan["chunks"]
    hdr = got[:4 * (-(-K // (16 * rpw))) * 16 * rpw * nch].reshape(-1, 16, rpw, nch, 4)
    return {(w, i): int(hdr[kt, w, i, 0, 3]) for w in range(16) for i in range(rpw)}


def reference_stream(host, plan, K, C, R, S, assign):
    """The documented layout, built directly from the CSR arrays for the
    given (wave, slot) -> row assignment of each channel tile."""
    rpw, cc, nch = plan["channels_per_wave"], plan["channels_per_chunk"], plan["chunks"]
    plp, vp, shift = plan["lds_channel_floats"], plan["lds_row_pitch"], plan["lds_col_shift"]
    kt_rows = 16 * rpw
    nkt = -(-K // kt_rows)
    rp, ci, va = host.rowptr, host.colidx, host.vals.view(np.int32)
    headers, entries = [], []
    for kt in range(nkt):
        k0 = kt * kt_rows
        slot = assign[kt]
        for w in range(16):
            for i in range(rpw):
                k = slot[(w, i)]
                for ch in range(nch):
                    start, counts = len(entries), [0, 0]
                    if k < K:
                        for parity in (0, 1):
                            for j in range(rp[k], rp[k + 1]):
                                c, t = divmod(int(ci[j]), R * S)
                                r, s = divmod(t, S)
                                if not ch * cc <= c < min(C, (ch + 1) * cc):
                                    continue
                                idx = (c - ch * cc) * plp + r * vp + s + shift
                                if idx % 2 != parity:
                                    continue
                                entries.append((idx - parity, int(va[j])))
                                counts[parity] += 1
                    headers.append((start, counts[0], counts[1], min(k, K)))
    out = np.array(headers, np.int32).reshape(-1)
    ent = np.array(entries + [(0, 0)] * 16, np.int32).reshape(-1)
    return np.concatenate([out, ent])


CASES = [
    # seed, N, C, K, H, W, pool, density, skew, unpadded
    (1, 2, 16, 40, 20, 20, False, 0.3, False, False),
    (2, 4, 64, 70, 30, 30, True, 0.2, True, False),
    (3, 2, 200, 33, 12, 12, False, 0.1, True, False),    # several chunks
    (4, 16, 3, 520, 12, 12, False, 0.3, True, False),    # four rows per wave
    (5, 8, 3, 520, 2, 2, False, 0.05, False, False),     # several images per tile
    (9, 32, 3, 1040, 2, 2, False, 0.05, False, False),   # four images, four rows per wave
    (6, 2, 24, 20, 16, 16, False, 0.3, False, True),     # unpadded input, rows of 16-byte groups
    (7, 1, 64, 64, 224, 224, False, 0.2, False, True),   # VGG-shaped, unpadded
    (8, 3, 5, 7, 9, 13, True, 0.5, False, False),        # odd widths
]


@pytest.mark.parametrize("case", CASES, ids=[f"c{c[0]}" for c in CASES])
def test_stream_matches_documented_layout(sp, case):
    seed, N, C, K, H, W, pool, d, skew, unpadded = case
    layer = synth.random_layer(7000 + seed, N, C, K, H, W, density=d, pool=pool, skew=skew)
    host = sp.spconv_pack_csr(layer.w, layer.mask, H + 2, W + 2)
    flags = sp.flags_of(True, pool) | (sp.SPCONV_UNPADDED_INPUT if unpadded else 0)
    mx = int(np.diff(host.rowptr).max())
    plan = sp.spconv_plan(N, C, H, W, sp.host_csr_struct(host), K, 3, 3, 1, 1, flags, max_row_nnz=mx)
    assert plan["kernel"] == sp.SPCONV_KERNEL_STRIDE1
    got = sp.spconv_pack_lowered(host, N, H, W, 1, 1, flags, mx)
    nkt = -(-K // (16 * plan["channels_per_wave"]))
    assign = [packed_slots(got, plan, K, kt) for kt in range(nkt)]
    for kt, slots in enumerate(assign):
        # every row of the tile in exactly one slot, the tile's padding rows empty (k = K)
        k0, kt_rows = kt * 16 * plan["channels_per_wave"], 16 * plan["channels_per_wave"]
        rows = sorted(slots.values())
        want = sorted(k if k < K else K for k in range(k0, k0 + kt_rows))
        assert rows == want
        # the balancing never does worse than the snake deal it starts from
        snake = {ws: (k if k < K else K) for ws, k in snake_slots(host, K, kt, plan["channels_per_wave"]).items()}
        assert chunk_costs(host, plan, K, C, 3, 3, slots) <= chunk_costs(host, plan, K, C, 3, 3, snake)
    ref = reference_stream(host, plan, K, C, 3, 3, assign)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)
    nh = -(-K // (16 * plan["channels_per_wave"])) * 16 * plan["channels_per_wave"] * plan["chunks"]
    assert got.size == 4 * nh + 2 * (host.nnz + 16)


def test_stream_plans_cover_the_interesting_tilings(sp):
    seen = set()
    for case in CASES:
        seed, N, C, K, H, W, pool, d, skew, unpadded = case
        layer = synth.random_layer(7000 + seed, N, C, K, H, W, density=d, pool=pool, skew=skew)
        host = sp.spconv_pack_csr(layer.w, layer.mask, H + 2, W + 2)
        flags = sp.flags_of(True, pool) | (sp.SPCONV_UNPADDED_INPUT if unpadded else 0)
        p = sp.spconv_plan(N, C, H, W, sp.host_csr_struct(host), K, 3, 3, 1, 1, flags,
                           max_row_nnz=int(np.diff(host.rowptr).max()))
        seen.add(("rpw", p["channels_per_wave"]))
        seen.add(("chunks>1", p["chunks"] > 1))
        seen.add(("ipw>1", p["images_per_group"] > 1))
        seen.add(("shift", p["lds_col_shift"] != 0))
        seen.add(("pitch!=Wp", p["lds_row_pitch"] != W + 2))
    for want in (("rpw", 1), ("rpw", 2), ("rpw", 4), ("chunks>1", True), ("ipw>1", True), ("shift", True),
                 ("pitch!=Wp", True)):
        assert want in seen, want


def test_pack_lowered_rejects_bad_input(sp):
    lib = sp._lib
    E = sp.SPCONV_EINVAL
    layer = synth.random_layer(7100, 2, 8, 12, 10, 10, density=0.4)
    host = sp.spconv_pack_csr(layer.w, layer.mask, 12, 12)
    opt = sp.spconv_options(0, 0, None, 0, None, 0)
    words = ctypes.c_int64()

    def size(N=2, C=8, H=10, W=10, K=12, stride=1, flags=1, st=None):
        st = sp.host_csr_struct(host) if st is None else st
        return lib.spconv_lowered_size(N, C, H, W, ctypes.byref(st), K, 3, 3, stride, 1, flags, ctypes.byref(opt),
                                       ctypes.byref(words))

    assert size() == sp.SPCONV_OK
    n = words.value
    buf = np.zeros(n, np.int32)

    def pack(st, cap=n):
        return lib.spconv_pack_lowered(2, 8, 10, 10, ctypes.byref(st), 12, 3, 3, 1, 1, 1, ctypes.byref(opt),
                                       buf.ctypes.data, cap)

    assert pack(sp.host_csr_struct(host)) == sp.SPCONV_OK
    assert pack(sp.host_csr_struct(host), n - 1) == sp.SPCONV_ECAPACITY
    assert lib.spconv_lowered_size(2, 8, 10, 10, ctypes.byref(sp.host_csr_struct(host)), 12, 3, 3, 1, 1, 1, None,
                                   None) == E
    assert lib.spconv_pack_lowered(2, 8, 10, 10, ctypes.byref(sp.host_csr_struct(host)), 12, 3, 3, 1, 1, 1, None,
                                   None, n) == E
    # the any-stride kernel takes no stream
    st2 = sp.spconv_csr(12, 8, 3, 3, 12, 12, host.nnz, host.rowptr.ctypes.data, host.colidx.ctypes.data,
                        host.offset.ctypes.data, host.vals.ctypes.data)
    assert size(stride=2, st=st2) == E
    # invalid CSR arrays
    for mutate in ("rowptr_decreasing", "rowptr_end", "col_range", "col_order"):
        bad = sp.HostCSR(host.K, host.C, host.R, host.S, host.Hp, host.Wp, host.rowptr.copy(), host.colidx.copy(),
                         host.offset.copy(), host.vals.copy())
        if mutate == "rowptr_decreasing":
            bad.rowptr[3] = bad.rowptr[4] + 1
        elif mutate == "rowptr_end":
            bad.rowptr[-1] -= 1
        elif mutate == "col_range":
            bad.colidx[5] = 8 * 9
        else:
            k = int(np.argmax(np.diff(bad.rowptr) >= 2))
            j = int(bad.rowptr[k])
            bad.colidx[j + 1] = bad.colidx[j]
        assert pack(sp.host_csr_struct(bad)) == E, mutate


def test_forward_checks_the_stream(sp):
    lib = sp._lib
    E = sp.SPCONV_EINVAL
    fake = 0x1000
    csr = sp.spconv_csr(4, 3, 3, 3, 10, 12, 5, fake, fake, fake, fake)
    opt = sp.spconv_options(0, 0, None, 0, None, 0)
    words = ctypes.c_int64()
    assert lib.spconv_lowered_size(2, 3, 8, 10, ctypes.byref(csr), 4, 3, 3, 1, 1, 1, ctypes.byref(opt),
                                   ctypes.byref(words)) == sp.SPCONV_OK

    def fwd(lowered, nwords, stride=1):
        o = sp.spconv_options(0, 0, None, 0, lowered, nwords)
        c = csr if stride == 1 else sp.spconv_csr(4, 3, 3, 3, 10, 12, 5, fake, fake, fake, fake)
        return lib.spconv_forward_ex(fake, 2, 3, 8, 10, ctypes.byref(c), 4, 3, 3, stride, 1, None, 1, ctypes.byref(o),
                                     fake, None)

    assert fwd(0x10000, words.value + 1) == E     # size of another plan
    assert fwd(0x10004, words.value) == E         # not 16-byte aligned
    assert fwd(0x10000, words.value, stride=2) == E


def _xcd_linear_id(b, G, xcds=8):
    """Workgroup id -> XCD-ordered index, as the kernels compute it (common.h)."""
    xcd, i = b % xcds, b // xcds
    per, rem = G // xcds, G % xcds
    return xcd * (per + 1) + i if xcd < rem else rem * (per + 1) + (xcd - rem) * per + i


@pytest.mark.parametrize("T", [1, 7, 255, 256, 257, 300, 511, 512, 528, 3584, 4864, 4999])
def test_persistent_schedule_takes_every_item_once(T):
    """The lowered kernel's workgroup b of a grid of G = min(T, 256) takes, at
    iteration t (while t*G + b < T), item t*G + its XCD-ordered index among
    that round's min(G, T - t*G) items: every item exactly once."""
    G = min(T, 256)
    seen = []
    for b in range(G):
        t = 0
        while t * G + b < T:
            seen.append(t * G + _xcd_linear_id(b, min(G, T - t * G)))
            t += 1
    assert sorted(seen) == list(range(T))


def _spanning_geometry_ok(Ho, Wo, vp, shift, R, S, PI, span, nt, PLp):
    """Row-spanning tiles as the stride-1 kernel indexes them: tile t starts at
    virtual pixel t*span of its image (row0 = that // vp, column phi), stages
    the window from column phi & ~3 of row0, and its lanes (64*PI tile pixels
    from phi) read window index (phi - col0) + q + r*vp + s + shift. Checks
    that the tiles' stored pixels are each output pixel once, that every read
    of every lane stays in [0, PLp), and that the rows whose column 0 falls in
    a tile (the side borders it zeroes) partition the rows."""
    cap = 64 * PI
    seen = np.zeros((Ho, Wo), np.int32)
    border_rows = np.zeros(Ho, np.int32)
    for t in range(nt):
        s0 = t * span
        row0 = s0 // vp
        phi = s0 - row0 * vp
        col0 = phi & ~3
        assert phi % 2 == 0 and (phi - col0) in (0, 2)
        q = np.arange(span)
        qa = q + phi
        y, x = row0 + qa // vp, qa % vp
        ok = (x < Wo) & (y < Ho)
        np.add.at(seen, (y[ok], x[ok]), 1)
        # the lowest read is an entry index (>= 0, odd taps stored rounded
        # down) plus phi - col0 >= 0; the highest the last lane's last tap
        hi = (phi - col0) + cap - 1 + (R - 1) * vp + (S - 1) + shift
        assert phi - col0 >= 0 and hi < PLp, (t, hi, PLp)
        r0 = row0 + (1 if phi > 0 else 0)
        r1 = min(-(-(row0 * vp + phi + span) // vp), Ho)
        border_rows[r0:max(r0, r1)] += 1
    assert np.all(seen == 1)
    assert np.all(border_rows == 1)


@pytest.mark.parametrize("seed", range(4))
def test_spanning_tiles_cover_each_pixel_once(seed):
    rng = np.random.default_rng(9300 + seed)
    for _ in range(60):
        PI = int(rng.choice([8, 12, 14, 16, 20, 24]))
        Wo = int(rng.integers(8, 300))
        Ho = int(rng.integers(2, 80))
        vp = Wo + 2 + int(rng.integers(0, 3))
        vp += vp & 1                                   # the planner requires an even pitch
        shift = int(rng.choice([0, 1, 2, 3]))
        span = 64 * PI - 2
        if Ho * vp <= 64 * PI - 1:
            continue                                   # whole-image tiles
        nt = -(-((Ho - 1) * vp + Wo) // span)
        PLp = -(-(shift + 3 + 64 * PI + 2 * vp + 3) // 4) * 4
        _spanning_geometry_ok(Ho, Wo, vp, shift, 3, 3, PI, span, nt, PLp)


def test_vgg_layer_plans_spanning_tiles_with_a_stream_only(sp):
    layer = synth.random_layer(9400, 32, 64, 64, 224, 224, density=0.2)
    host = sp.spconv_pack_csr(layer.w, layer.mask, 226, 226)
    st = sp.host_csr_struct(host)
    mx = int(np.diff(host.rowptr).max())
    for flags in (sp.flags_of(True, False), sp.flags_of(True, False) | sp.SPCONV_UNPADDED_INPUT):
        p = sp.spconv_plan(32, 64, 224, 224, st, 64, 3, 3, 1, 1, flags, max_row_nnz=mx, lowered=True)
        plain = sp.spconv_plan(32, 64, 224, 224, st, 64, 3, 3, 1, 1, flags, max_row_nnz=mx)
        assert plain["tile_pixels"] == 0
        assert (p["pixels_per_lane"], p["channels_per_wave"]) == (plain["pixels_per_lane"], plain["channels_per_wave"])
        span, vp = p["tile_pixels"], p["lds_row_pitch"]
        assert span == 64 * p["pixels_per_lane"] - 2
        assert p["tiles_per_image"] == -(-(223 * vp + 224) // span)
        _spanning_geometry_ok(224, 224, vp, p["lds_col_shift"], 3, 3, p["pixels_per_lane"], span,
                              p["tiles_per_image"], p["lds_channel_floats"])
        # the stream for this plan, word for word
        got = sp.spconv_pack_lowered(host, 32, 224, 224, 1, 1, flags, mx)
        nkt = -(-64 // (16 * p["channels_per_wave"]))
        assign = [packed_slots(got, p, 64, kt) for kt in range(nkt)]
        assert np.array_equal(got, reference_stream(host, p, 64, 64, 3, 3, assign))
    # pooled layers keep whole-row tiles
    pooled = sp.spconv_plan(32, 64, 224, 224, st, 64, 3, 3, 1, 1, sp.flags_of(True, True), max_row_nnz=mx,
                            lowered=True)
    assert pooled["tile_pixels"] == 0


@pytest.mark.parametrize("case", CASES, ids=[f"c{c[0]}" for c in CASES])
def test_plans_reserve_the_prefetch_sink(sp, case):
    # The walk's entry-stream prefetch lands in 64 floats after everything else
    # the stride-1 kernel keeps in LDS: the plan's dynamic LDS must hold the two
    # chunk buffers (or the pooled staging) plus that sink, within 160 KiB.
    seed, N, C, K, H, W, pool, d, skew, unpadded = case
    layer = synth.random_layer(7000 + seed, N, C, K, H, W, density=d, pool=pool, skew=skew)
    host = sp.spconv_pack_csr(layer.w, layer.mask, H + 2, W + 2)
    flags = sp.flags_of(True, pool) | (sp.SPCONV_UNPADDED_INPUT if unpadded else 0)
    for lowered in (False, True):
        p = sp.spconv_plan(N, C, H, W, sp.host_csr_struct(host), K, 3, 3, 1, 1, flags,
                           max_row_nnz=int(np.diff(host.rowptr).max()), lowered=lowered)
        assert p["kernel"] == sp.SPCONV_KERNEL_STRIDE1
        buf = -(-p["images_per_group"] * p["channels_per_chunk"] * p["lds_channel_floats"] // 64) * 64
        need = 2 * buf
        if pool:
            need = max(need, 16 * p["images_per_group"] * 64 * p["pixels_per_lane"])
        assert p["lds_bytes"] >= 4 * (need + 64)
        assert p["lds_bytes"] <= 160 * 1024


def test_packer_gives_older_waves_more_entries(sp):
    # Waves w, w+4, w+8, w+12 share a SIMD, which issues the oldest ready wave
    # first; the packer weights each wave's entries by its age share, so on a
    # VGG-shaped layer the oldest quarter of the waves carries more entries per
    # chunk than the youngest, while each SIMD's total stays balanced.
    layer = synth.random_layer(9401, 32, 64, 64, 224, 224, density=0.2)
    host = sp.spconv_pack_csr(layer.w, layer.mask, 226, 226)
    mx = int(np.diff(host.rowptr).max())
    flags = sp.flags_of(True, False)
    p = sp.spconv_plan(32, 64, 224, 224, sp.host_csr_struct(host), 64, 3, 3, 1, 1, flags, max_row_nnz=mx,
                       lowered=True)
    got = sp.spconv_pack_lowered(host, 32, 224, 224, 1, 1, flags, mx)
    rpw, nch = p["channels_per_wave"], p["chunks"]
    nkt = -(-64 // (16 * rpw))
    hdr = got[:4 * nkt * 16 * rpw * nch].reshape(nkt, 16, rpw, nch, 4)
    load = (hdr[..., 1] + hdr[..., 2]).sum(axis=2)          # (tile, wave, chunk)
    group = load.reshape(nkt, 4, 4, nch).mean(axis=(0, 2, 3))  # by age group (wave // 4)
    assert group[0] > group[3] * 1.08
    simd = load.reshape(nkt, 4, 4, nch).sum(axis=1)          # (tile, simd, chunk)
    assert (simd.max(axis=1) / simd.mean(axis=1)).mean() < 1.08
