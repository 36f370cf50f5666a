"""The kernel-instance case table covers exactly what the library compiles,
and every case still makes the planner pick its instance (host only: the
plans read no device memory). A new instance without a case, or a planner
change that moves a case to another instance, fails here before any GPU run."""
import pytest

import variant_cases as vc
from paper_2005_04091_amd import spconv as sp


def test_table_covers_every_compiled_instance():
    s1 = set(sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1))
    dense = set(sp.spconv_kernel_variants(sp.SPCONV_KERNEL_DENSE))
    assert len(s1) == len(sp.spconv_kernel_variants(sp.SPCONV_KERNEL_STRIDE1))
    have_s1 = {c[1] for c in vc.CASES if c[0] == "s1"}
    have_dense = {c[1] for c in vc.CASES if c[0] == "dense"}
    assert have_s1 == s1, f"missing {sorted(s1 - have_s1)}, stale {sorted(have_s1 - s1)}"
    assert have_dense == dense, f"missing {sorted(dense - have_dense)}, stale {sorted(have_dense - dense)}"
    assert all(len(c) == 11 for c in vc.CASES), "a case without a shape"


@pytest.mark.parametrize("case", vc.CASES, ids=[f"{c[0]}{c[1]}" for c in vc.CASES])
def test_case_plans_to_its_instance(case):
    assert vc.planned_variant(case) == case[1]


def test_cases_are_small():
    """Each case is a few hundred million multiply-adds of oracle work at most."""
    assert max(vc.oracle_cost(c) for c in vc.CASES) < 3e8
    assert sum(vc.oracle_cost(c) for c in vc.CASES) < 3e9


def test_generic_kernel_instances():
    assert sp.spconv_kernel_variants(sp.SPCONV_KERNEL_GENERIC) == [(4, 0, 4, 0), (4, 0, 4, 1)]
    with pytest.raises(sp.SpconvError):
        sp.spconv_kernel_variants(99)
