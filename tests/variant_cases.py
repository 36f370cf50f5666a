"""One small layer per compiled kernel instance, for the GPU parity tests.

Every (pixels per lane, images per group, channels per wave, pool) instance of
the stride-1 sparse kernel and every (R, S, pixel blocks per wave, pool)
instance of the dense kernel that the library compiles (``spconv_kernel_variants``)
has a case here: a seeded synthetic layer (``synth.random_layer``) on which the
library's own planner picks that instance. ``tests/test_variants_cpu.py`` checks
on the CPU that the table covers exactly the compiled instances and that each
case still plans to its instance; ``tests/test_gpu_variants.py`` runs every case
on the GPU against the oracle over whole output tensors.

When the tilings or the planners change, ``python tests/variant_cases.py``
searches the shapes again (planner calls only, on host-side CSR structs whose
arrays are never read) and prints a new table to paste below.
"""
from __future__ import annotations

import sys
from pathlib import Path

ROOT = Path(__file__).resolve().parent.parent
if str(ROOT) not in sys.path:
    sys.path.insert(0, str(ROOT))

# (kind, variant, N, C, K, H, W, density, skew, pool, seed); kind "s1" = stride-1
# sparse kernel, variant (PI, IPW, RPW, pool); "s1t" = the same kernel run with
# a lowered stream on more work items than one round of workgroups (the tiled
# form); kind "dense", variant (R, S, NB, pool).
CASES = [
    ('s1', (24, 1, 1, 0), 1, 3, 1040, 64, 64, 0.8, False, False, 5000),
    ('s1', (24, 1, 1, 1), 1, 3, 1040, 64, 64, 0.05, False, True, 5100),
    ('s1', (22, 1, 1, 0), 16, 3, 256, 36, 36, 0.8, False, False, 5200),
    ('s1', (22, 1, 1, 1), 2, 3, 1040, 36, 36, 0.05, False, True, 5300),
    ('s1', (20, 1, 1, 0), 128, 3, 16, 48, 48, 0.05, False, False, 5400),
    ('s1', (20, 1, 1, 1), 1, 3, 1040, 56, 56, 0.05, False, True, 5500),
    ('s1', (18, 1, 1, 0), 64, 3, 16, 64, 64, 0.05, False, False, 5600),
    ('s1', (18, 1, 1, 1), 2, 3, 1040, 32, 32, 0.05, False, True, 5700),
    ('s1', (16, 1, 1, 0), 4, 3, 16, 224, 224, 0.05, True, False, 5800),
    ('s1', (16, 1, 1, 1), 2, 3, 1040, 29, 29, 0.05, False, True, 5900),
    ('s1', (14, 1, 1, 0), 64, 3, 16, 56, 56, 0.05, True, False, 6000),
    ('s1', (14, 1, 1, 1), 2, 3, 1040, 27, 27, 0.05, False, True, 6100),
    ('s1', (12, 1, 1, 0), 128, 3, 16, 36, 36, 0.05, True, False, 6200),
    ('s1', (12, 1, 1, 1), 2, 3, 1040, 25, 25, 0.05, False, True, 6300),
    ('s1', (10, 1, 1, 0), 128, 3, 16, 31, 31, 0.05, True, False, 6400),
    ('s1', (10, 1, 1, 1), 2, 3, 1040, 22, 22, 0.05, False, True, 6500),
    ('s1', (8, 1, 1, 0), 128, 3, 16, 27, 27, 0.05, True, False, 6600),
    ('s1', (8, 1, 1, 1), 2, 3, 1040, 19, 19, 0.05, False, True, 6700),
    ('s1', (6, 1, 1, 0), 64, 3, 16, 30, 30, 0.05, True, False, 6800),
    ('s1', (6, 1, 1, 1), 2, 3, 1040, 16, 16, 0.05, False, True, 6900),
    ('s1', (4, 1, 1, 0), 1, 3, 16, 2, 2, 0.05, True, False, 7000),
    ('s1', (4, 1, 1, 1), 1, 3, 16, 2, 2, 0.05, False, True, 7100),
    ('s1', (16, 1, 2, 0), 32, 3, 256, 31, 31, 0.05, False, False, 7200),
    ('s1', (16, 1, 2, 1), 4, 3, 1040, 29, 29, 0.05, False, True, 7300),
    ('s1', (14, 1, 2, 0), 32, 3, 256, 27, 27, 0.2, False, False, 7400),
    ('s1', (14, 1, 2, 1), 4, 3, 1040, 27, 27, 0.05, False, True, 7500),
    ('s1', (12, 1, 2, 0), 1, 3, 1040, 64, 64, 0.3, False, False, 7600),
    ('s1', (12, 1, 2, 1), 4, 3, 1040, 25, 25, 0.05, False, True, 7700),
    ('s1', (10, 1, 2, 0), 16, 3, 256, 31, 31, 0.2, False, False, 7800),
    ('s1', (10, 1, 2, 1), 4, 3, 1040, 22, 22, 0.05, False, True, 7900),
    ('s1', (8, 1, 2, 0), 16, 3, 256, 30, 30, 0.05, False, False, 8000),
    ('s1', (8, 1, 2, 1), 2, 16, 1040, 36, 36, 0.05, False, True, 8100),
    ('s1', (6, 1, 2, 0), 8, 3, 520, 16, 16, 0.05, False, False, 8200),
    ('s1', (6, 1, 2, 1), 4, 32, 1040, 18, 18, 0.05, True, True, 8300),
    ('s1', (4, 1, 2, 0), 32, 3, 256, 2, 2, 0.05, False, False, 8400),
    ('s1', (4, 1, 2, 1), 4, 64, 1040, 11, 11, 0.05, True, True, 8500),
    ('s1', (8, 1, 4, 0), 8, 3, 1040, 19, 19, 0.05, False, False, 8600),
    ('s1', (8, 1, 4, 1), 4, 16, 1040, 36, 36, 0.05, False, True, 8700),
    ('s1', (6, 1, 4, 0), 8, 3, 1040, 16, 16, 0.05, False, False, 8800),
    ('s1', (6, 1, 4, 1), 4, 64, 1040, 29, 29, 0.05, True, True, 8900),
    ('s1', (4, 1, 4, 0), 8, 3, 1040, 11, 11, 0.05, False, False, 9000),
    ('s1', (4, 1, 4, 1), 4, 32, 1040, 22, 22, 0.3, True, True, 9100),
    ('s1', (8, 2, 1, 0), 4, 3, 1040, 19, 19, 0.8, False, False, 9200),
    ('s1', (8, 2, 1, 1), 4, 3, 1040, 19, 19, 0.05, False, True, 9300),
    ('s1', (6, 2, 1, 0), 4, 3, 1040, 16, 16, 0.8, False, False, 9400),
    ('s1', (6, 2, 1, 1), 4, 3, 1040, 16, 16, 0.05, False, True, 9500),
    ('s1', (4, 2, 1, 0), 4, 3, 1040, 11, 11, 0.8, False, False, 9600),
    ('s1', (4, 2, 1, 1), 4, 3, 1040, 11, 11, 0.05, False, True, 9700),
    ('s1', (2, 2, 1, 0), 8, 3, 520, 2, 2, 0.05, False, False, 9802),
    ('s1', (2, 2, 1, 1), 4, 3, 1040, 2, 2, 0.05, False, True, 9900),
    ('s1', (8, 2, 2, 0), 8, 3, 1040, 19, 19, 0.3, False, False, 10000),
    ('s1', (8, 2, 2, 1), 8, 3, 1040, 19, 19, 0.05, False, True, 10100),
    ('s1', (6, 2, 2, 0), 8, 3, 1040, 16, 16, 0.3, False, False, 10200),
    ('s1', (6, 2, 2, 1), 8, 32, 1040, 16, 16, 0.05, False, True, 10300),
    ('s1', (4, 2, 2, 0), 8, 3, 1040, 11, 11, 0.2, False, False, 10404),
    ('s1', (4, 2, 2, 1), 8, 32, 1040, 11, 11, 0.05, True, True, 10500),
    ('s1', (2, 2, 2, 0), 8, 3, 1040, 2, 2, 0.05, False, False, 10600),
    ('s1', (2, 2, 2, 1), 8, 16, 1040, 2, 2, 0.3, True, True, 10700),
    ('s1', (4, 2, 4, 0), 16, 3, 1040, 11, 11, 0.05, False, False, 10800),
    ('s1', (4, 2, 4, 1), 16, 250, 1040, 11, 11, 0.05, True, True, 10900),
    ('s1', (2, 2, 4, 0), 16, 3, 1040, 2, 2, 0.05, False, False, 11000),
    ('s1', (2, 2, 4, 1), 16, 250, 1040, 2, 2, 0.2, True, True, 11100),
    ('s1', (6, 4, 1, 0), 8, 3, 1040, 16, 16, 0.8, False, False, 11200),
    ('s1', (6, 4, 1, 1), 8, 3, 1040, 16, 16, 0.05, False, True, 11300),
    ('s1', (4, 4, 1, 0), 8, 3, 1040, 11, 11, 0.8, False, False, 11400),
    ('s1', (4, 4, 1, 1), 8, 3, 1040, 11, 11, 0.05, False, True, 11500),
    ('s1', (2, 4, 1, 0), 8, 3, 1040, 2, 2, 0.8, False, False, 11600),
    ('s1', (2, 4, 1, 1), 8, 3, 1040, 2, 2, 0.05, False, True, 11700),
    ('s1', (4, 4, 2, 0), 16, 3, 1040, 11, 11, 0.3, False, False, 11802),
    ('s1', (4, 4, 2, 1), 16, 3, 1040, 11, 11, 0.05, False, True, 11900),
    ('s1', (2, 4, 2, 0), 16, 3, 1040, 2, 2, 0.2, False, False, 12003),
    ('s1', (2, 4, 2, 1), 16, 3, 1040, 2, 2, 0.05, False, True, 12100),
    ('s1', (2, 4, 4, 0), 32, 3, 1040, 2, 2, 0.05, False, False, 12200),
    ('s1', (2, 4, 4, 1), 32, 3, 1040, 2, 2, 0.2, True, True, 12300),
    ('s1t', (24, 1, 1, 0), 16, 3, 256, 64, 64, 0.8, False, False, 12400),
    ('s1t', (24, 1, 1, 1), 2, 3, 1040, 64, 64, 0.05, False, True, 12500),
    ('s1t', (22, 1, 1, 0), 32, 3, 256, 36, 36, 0.8, False, False, 12600),
    ('s1t', (22, 1, 1, 1), 4, 3, 1040, 36, 36, 0.05, False, True, 12707),
    ('s1t', (20, 1, 1, 0), 16, 3, 256, 48, 48, 0.8, False, False, 12800),
    ('s1t', (20, 1, 1, 1), 2, 3, 1040, 56, 56, 0.05, False, True, 12901),
    ('s1t', (18, 1, 1, 0), 128, 3, 16, 64, 64, 0.05, False, False, 13000),
    ('s1t', (18, 1, 1, 1), 4, 3, 1040, 32, 32, 0.05, False, True, 13100),
    ('s1t', (16, 1, 1, 0), 8, 3, 16, 224, 224, 0.05, True, False, 13200),
    ('s1t', (16, 1, 1, 1), 32, 3, 16, 112, 112, 0.05, False, True, 13300),
    ('s1t', (14, 1, 1, 0), 128, 3, 16, 56, 56, 0.05, True, False, 13400),
    ('s1t', (14, 1, 1, 1), 128, 3, 16, 56, 56, 0.05, False, True, 13500),
    ('s1t', (12, 1, 1, 0), 16, 3, 1040, 25, 25, 0.8, False, False, 13600),
    ('s1t', (12, 1, 1, 1), 8, 3, 1040, 25, 25, 0.5, False, True, 13700),
    ('s1t', (16, 1, 2, 0), 8, 3, 16, 224, 224, 0.05, False, False, 13806),
    ('s1t', (16, 1, 2, 1), 64, 3, 256, 29, 29, 0.05, False, True, 13900),
    ('s1t', (14, 1, 2, 0), 64, 3, 256, 27, 27, 0.2, False, False, 14000),
    ('s1t', (14, 1, 2, 1), 64, 3, 256, 27, 27, 0.05, False, True, 14100),
    ('s1t', (12, 1, 2, 0), 16, 3, 256, 64, 64, 0.05, True, False, 14200),
    ('s1t', (12, 1, 2, 1), 64, 3, 256, 25, 25, 0.05, False, True, 14300),
    ('dense', (3, 3, 1, 0), 1, 3, 16, 2, 2, 0.3, False, False, 14400),
    ('dense', (3, 3, 1, 1), 1, 3, 16, 2, 2, 0.3, False, True, 14500),
    ('dense', (3, 3, 2, 0), 1, 3, 16, 31, 31, 0.3, False, False, 14600),
    ('dense', (3, 3, 2, 1), 1, 3, 16, 15, 15, 0.3, False, True, 14700),
    ('dense', (3, 3, 3, 0), 1, 3, 16, 64, 64, 0.3, False, False, 14800),
    ('dense', (3, 3, 3, 1), 1, 3, 16, 31, 31, 0.3, False, True, 14900),
    ('dense', (3, 3, 4, 0), 1, 3, 16, 112, 112, 0.3, False, False, 15000),
    ('dense', (3, 3, 4, 1), 1, 3, 16, 48, 48, 0.3, False, True, 15100),
    ('dense', (3, 3, 5, 0), 128, 3, 16, 29, 29, 0.3, False, False, 15200),
    ('dense', (3, 3, 5, 1), 1, 3, 16, 64, 64, 0.3, False, True, 15300),
    ('dense', (3, 3, 6, 0), 128, 3, 64, 21, 21, 0.3, False, False, 15400),
    ('dense', (3, 3, 6, 1), 1, 3, 16, 80, 80, 0.3, False, True, 15500),
    ('dense', (3, 3, 7, 0), 64, 3, 16, 64, 64, 0.3, False, False, 15600),
    ('dense', (3, 3, 7, 1), 64, 3, 16, 48, 48, 0.3, False, True, 15700),
    ('dense', (3, 3, 8, 0), 1, 3, 16, 224, 224, 0.3, False, False, 15800),
    ('dense', (3, 3, 8, 1), 1, 3, 16, 112, 112, 0.3, False, True, 15900),
    ('dense', (1, 1, 1, 0), 1, 3, 16, 2, 2, 0.3, False, False, 16000),
    ('dense', (1, 1, 1, 1), 1, 3, 16, 2, 2, 0.3, False, True, 16100),
    ('dense', (1, 1, 2, 0), 1, 3, 16, 36, 36, 0.3, False, False, 16200),
    ('dense', (1, 1, 2, 1), 1, 3, 16, 17, 17, 0.3, False, True, 16300),
    ('dense', (1, 1, 3, 0), 1, 3, 16, 80, 80, 0.3, False, False, 16400),
    ('dense', (1, 1, 3, 1), 1, 3, 16, 36, 36, 0.3, False, True, 16500),
    ('dense', (1, 1, 4, 0), 1, 3, 16, 112, 112, 0.3, False, False, 16600),
    ('dense', (1, 1, 4, 1), 1, 3, 16, 56, 56, 0.3, False, True, 16700),
    ('dense', (1, 1, 5, 0), 128, 3, 16, 29, 29, 0.3, False, False, 16800),
    ('dense', (1, 1, 5, 1), 1, 3, 16, 80, 80, 0.3, False, True, 16900),
    ('dense', (1, 1, 6, 0), 64, 3, 16, 48, 48, 0.3, False, False, 17000),
    ('dense', (1, 1, 6, 1), 64, 3, 16, 48, 48, 0.3, False, True, 17100),
    ('dense', (1, 1, 7, 0), 1, 3, 16, 224, 224, 0.3, False, False, 17200),
    ('dense', (1, 1, 7, 1), 1, 3, 16, 112, 112, 0.3, False, True, 17300),
    ('dense', (1, 1, 8, 0), 64, 3, 16, 64, 64, 0.3, False, False, 17400),
    ('dense', (1, 1, 8, 1), 64, 3, 16, 64, 64, 0.3, False, True, 17500),
]

# Shapes the search tries (small enough that the oracle finishes in well under
# a second per case at the chosen one).
_SEARCH_H = list(range(2, 33)) + [36, 40, 48, 56, 64, 80, 112, 224]
_SEARCH_N = (1, 2, 4, 8, 16, 32, 64, 128)
_SEARCH_C = (3, 16, 32, 64, 250)
_SEARCH_K = (16, 64, 128, 256, 520, 1040)


def case_layer(case):
    """The seeded synthetic layer of one case."""
    from paper_2005_04091_amd import synth
    kind, variant, N, C, K, H, W, d, skew, pool, seed = case
    R = S = variant[0] if kind == "dense" else 3
    pad = (R - 1) // 2
    return synth.random_layer(seed, N, C, K, H, W, R, S, 1, pad, d, True, pool, True, skew)


def planned_variant(case, layer=None):
    """The instance the library's planner picks for this case's layer (host
    only: the CSR is packed on the host and the plan reads no array)."""
    import numpy as np
    from paper_2005_04091_amd import spconv as sp
    kind, variant, N, C, K, H, W, d, skew, pool, seed = case
    layer = case_layer(case) if layer is None else layer
    R, S = layer.w.shape[2], layer.w.shape[3]
    flags = sp.flags_of(True, pool)
    if kind == "dense":
        p = sp.spconv_dense_plan(N, C, H, W, K, R, S, layer.pad, flags)
        return (R, S, p["pixels_per_lane"], int(pool))
    host = sp.spconv_pack_csr(layer.w, layer.mask, H + 2 * layer.pad, W + 2 * layer.pad)
    mx = int(np.diff(host.rowptr).max())
    p = sp.spconv_plan(N, C, H, W, sp.host_csr_struct(host), K, R, S, 1, layer.pad, flags, max_row_nnz=mx,
                       lowered=True)
    if p["kernel"] != sp.SPCONV_KERNEL_STRIDE1:
        return None
    # "s1t": the lowered launch runs several work items per workgroup
    if (kind == "s1t") != (p["launch_workgroups"] < p["workgroups"]):
        return None
    return (p["pixels_per_lane"], p["images_per_group"], p["channels_per_wave"], int(pool))


def oracle_cost(case):
    """Multiply-adds the oracle spends on a case (its nonzeros x output pixels)."""
    kind, variant, N, C, K, H, W, d, skew, pool, seed = case
    taps = variant[0] * variant[1] if kind == "dense" else 9
    return N * K * H * W * max(1.0, d * C * taps)


def search():
    """Cheapest verified case per compiled instance (see the module docstring)."""
    import numpy as np
    from paper_2005_04091_amd import spconv as sp
    dummy = np.zeros(4, np.int32)
    ptr = dummy.ctypes.data
    tiled = set(sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1_TILED))
    cands = {}
    for H in _SEARCH_H:
        for N in _SEARCH_N:
            for C in _SEARCH_C:
                for K in _SEARCH_K:
                    for pool in (False, True):
                        for d in (0.05, 0.2, 0.3, 0.5, 0.8):
                            nnz = max(1, int(d * K * C * 9))
                            for skew in (False, True):
                                # The hint the binding will pass: the largest row of the
                                # drawn filter (binomial spread for uniform rows, about 2.6x
                                # the mean for Beta(2, 5) rows).
                                mean = nnz / K
                                mx = 2.6 * mean if skew else mean + 3.5 * (mean * (1 - d)) ** 0.5
                                mx = min(nnz, int(mx))
                                st = sp.spconv_csr(K, C, 3, 3, H + 2, H + 2, nnz, ptr, ptr, ptr, ptr)
                                try:
                                    p = sp.spconv_plan(N, C, H, H, st, K, 3, 3, 1, 1, sp.flags_of(True, pool),
                                                       max_row_nnz=mx)
                                except sp.SpconvError:
                                    continue
                                if p["kernel"] != sp.SPCONV_KERNEL_STRIDE1:
                                    continue
                                v = (p["pixels_per_lane"], p["images_per_group"], p["channels_per_wave"], int(pool))
                                kind = "s1t" if p["workgroups"] > 256 and v in tiled else "s1"
                                cands.setdefault((kind, v), []).append((kind, v, N, C, K, H, H, d, skew, pool, 0))
                        for rs in (3, 1):
                            try:
                                p = sp.spconv_dense_plan(N, C, H, H, K, rs, rs, (rs - 1) // 2,
                                                         sp.flags_of(True, pool))
                            except sp.SpconvError:
                                continue
                            v = (rs, rs, p["pixels_per_lane"], int(pool))
                            cands.setdefault(("dense", v), []).append(("dense", v, N, C, K, H, H, 0.3, False, pool, 0))
    table = []
    wanted = [("s1", v) for v in sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1)] + \
             [("s1t", v) for v in sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1_TILED)] + \
             [("dense", v) for v in sp.spconv_kernel_variants(sp.SPCONV_KERNEL_DENSE)]
    for kind, v in wanted:
        got = None
        pool_of = cands.get((kind, v), []) + (cands.get(("s1t", v), []) if kind == "s1" else [])
        for c in sorted(pool_of, key=oracle_cost):
            _, _, N, C, K, H, W = c[:7]
            if N * C * H * W > 4_000_000 or K * C * 9 > 4_000_000:
                continue  # too large to draw for a test case
            for seed in range(5000 + 100 * len(table), 5000 + 100 * len(table) + 8):
                case = (kind,) + c[1:-1] + (seed,)
                if planned_variant(case) == v:
                    got = case
                    break
            if got:
                break
        table.append(got if got else (kind, v, None))
    return table


if __name__ == "__main__":
    for case in search():
        print(f"    {case!r},")
