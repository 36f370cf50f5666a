"""The stride-1 kernel's staging of an unpadded input, as index arithmetic on
the CPU (no GPU needed).

The kernel copies each channel chunk in blocks of consecutive LDS floats (64
lanes of 4 or 16 bytes); a lane maps its LDS position to (channel slot, staged
row, image column) with two multiply-shift divisions and reads either the
image pixel there or, through an offset past the buffer's range, a zero. This
test runs that map, written as the kernel computes it, over random layer
shapes, pads, tile positions and chunk sizes, and checks that every position of
the chunk's slots receives the value of the zero-padded layout (image pixel,
border or gap zero), that every read stays inside the buffer range, and that a
16-byte lane never straddles the image row's edge.
"""
import random

import pytest


def _div_magic(d):
    """Round-up reciprocal for x // d with x < 2^31 (the kernels' fast_div)."""
    if d == 1:
        return 1, 0
    L = 0
    while (1 << L) < d:
        L += 1
    s = 31 + L
    return ((1 << s) + d - 1) // d, s


def _staged(W, H, pad, R, TH, C, Cc, ch, ty, dma16):
    """Per LDS position of the chunk's slots: what the staging writes there."""
    Hp, Wp = H + 2 * pad, W + 2 * pad
    row16 = W % 4 == 0
    vp = (Wp + 3) // 4 * 4 if row16 else Wp
    shift = (4 - pad % 4) % 4 if row16 else 0
    rows_in = TH + R - 1
    PLp = (rows_in * vp + shift + 3) // 4 * 4
    c0 = ch * Cc
    cn = min(Cc, C - c0)
    in_row0 = ty * TH
    per_lane = 4 if dma16 else 1
    span = cn * PLp
    y_lo = max(in_row0 - pad, 0)
    y_span = max(min(in_row0 - pad + rows_in, H) - y_lo, 0)
    nrec = ((cn - 1) * H + y_span) * W * 4
    lead = shift + pad
    pm, ps = _div_magic(PLp)
    vm, vs = _div_magic(vp)
    got = {}
    for b in range((span + 64 * per_lane - 1) // (64 * per_lane)):
        for lane in range(64):
            P = b * 64 * per_lane + lane * per_lane
            if P >= span:
                continue
            cl = (P * pm) >> ps
            t = P - cl * PLp - lead
            assert t + vp >= 0
            i = ((t + vp) * vm >> vs) - 1
            x = t - i * vp
            y = in_row0 + i - pad
            if i < rows_in and x < W and 0 <= y < H:
                voff = ((cl * H + (y - y_lo)) * W + x) * 4
                assert 0 <= voff and voff + 4 * per_lane <= nrec
                assert x + per_lane <= W
                for e in range(per_lane):
                    got[P + e] = (c0 + cl, y, x + e)
            else:
                for e in range(per_lane):
                    got[P + e] = 0
    assert nrec < 2 ** 32
    return got, (span, PLp, vp, shift, rows_in, in_row0, c0)


@pytest.mark.parametrize("seed", range(8))
def test_unpadded_staging_writes_the_padded_layout(seed):
    rng = random.Random(9100 + seed)
    done = 0
    while done < 120:
        W = rng.choice([1, 2, 3, 4, 5, 7, 8, 12, 14, 16, 28, 56, 60, 224, 225])
        H = rng.randint(1, 30)
        pad = rng.choice([0, 1, 1, 2, 3, 4, 5])
        R = rng.choice([1, 3, 3, 5])
        if H + 2 * pad < R:
            continue
        Ho = H + 2 * pad - R + 1
        TH = rng.randint(1, Ho)
        C = rng.randint(1, 5)
        Cc = rng.randint(1, C)
        ch = rng.randint(0, (C - 1) // Cc)
        ty = rng.randint(0, (Ho - 1) // TH)
        dma16 = W % 4 == 0 and rng.random() < 0.8
        got, (span, PLp, vp, shift, rows_in, in_row0, c0) = _staged(W, H, pad, R, TH, C, Cc, ch, ty, dma16)
        Wp = W + 2 * pad
        for P in range(span):
            cl, rem = divmod(P, PLp)
            want = 0
            if rem >= shift:
                i, j = divmod(rem - shift, vp)
                x, y = j - pad, in_row0 + i - pad
                if i < rows_in and j < Wp and 0 <= x < W and 0 <= y < H:
                    want = (c0 + cl, y, x)
            assert got.get(P) == want, (W, H, pad, R, TH, C, Cc, ch, ty, dma16, P)
        done += 1


def test_unit_walk_visits_every_unit_once():
    """The staging loops deal units u = q*n + r to `step` waves without a
    division per unit: wave w starts at q = (w * ceil(2^16/n)) >> 16, r = w -
    q*n, and advances by q += step // n, r += step % n with one wrap. For every
    slot width n a plan can have (channel slots of up to 160 blocks, rows of up
    to 40) and every wave count, each wave visits exactly u = w, w + step, ..."""
    for step in (1, 4, 8, 12, 16):
        for n in range(1, 161):
            recip = (65536 + n - 1) // n
            dq, dr = divmod(step, n)
            total = 7 * n + 3
            seen = []
            for w in range(step):
                q = (w * recip) >> 16
                r = w - q * n
                assert (q, r) == divmod(w, n)
                u = w
                while q * n + r < total:
                    assert q * n + r == u and 0 <= r < n
                    seen.append(u)
                    q += dq
                    r += dr
                    if r >= n:
                        r -= n
                        q += 1
                    u += step
            assert sorted(seen) == list(range(total))
