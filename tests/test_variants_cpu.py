"""The kernel-instance case table covers exactly what the library compiles,
and every case still makes the planner pick its instance (host only: the
plans read no device memory). A new instance without a case, or a planner
change that moves a case to another instance, fails here before any GPU run."""
import pytest

import variant_cases as vc
from paper_2005_04091_amd import spconv as sp


def test_table_covers_every_compiled_instance():
    for kind, family in (("s1", sp.SPCONV_KERNEL_STRIDE1), ("s1t", sp.SPCONV_KERNEL_STRIDE1_TILED),
                         ("dense", sp.SPCONV_KERNEL_DENSE)):
        compiled = sp.spconv_kernel_variants(family)
        assert len(set(compiled)) == len(compiled)
        have = {c[1] for c in vc.CASES if c[0] == kind}
        assert have == set(compiled), f"{kind}: missing {sorted(set(compiled) - have)}, stale {sorted(have - set(compiled))}"
    # the tiled form exists for a subset of the stride-1 tilings
    assert set(sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1_TILED)) <= \
        set(sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1))
    assert all(len(c) == 11 for c in vc.CASES), "a case without a shape"


@pytest.mark.parametrize("case", vc.CASES, ids=[f"{c[0]}{c[1]}" for c in vc.CASES])
def test_case_plans_to_its_instance(case):
    assert vc.planned_variant(case) == case[1]


def test_cases_are_small():
    """Each case is a few hundred million multiply-adds of oracle work at most."""
    assert max(vc.oracle_cost(c) for c in vc.CASES) < 4e8
    assert sum(vc.oracle_cost(c) for c in vc.CASES) < 3e9


def test_generic_kernel_instances():
    assert sp.spconv_kernel_variants(sp.SPCONV_KERNEL_GENERIC) == [(4, 0, 4, 0), (4, 0, 4, 1)]
    with pytest.raises(sp.SpconvError):
        sp.spconv_kernel_variants(99)
