"""Host side of the polynomial-set search: the candidate sets for F(m x m, 3x3)
have the right degree sums, are valid plans (built by the library on the
CPU), and fall inside the compiled kernel shapes."""
import pytest

from paper_1905_05233_amd import search as S
from paper_1905_05233_amd.winograd import Plan


def _degree(mod):
    if mod == "inf":
        return 1
    if "a^3" in mod:
        return 3
    if "a^2" in mod:
        return 2
    return 1


@pytest.mark.parametrize("m", [2, 4, 6, 8])
def test_candidate_sets_are_valid_plans(m):
    sets = S.candidate_sets(m, max_quadratic=2)
    assert len(sets) == len(set(sets))
    for spec in sets:
        mods = spec.split(",")
        assert sum(_degree(x) for x in mods) == m + 2          # m + r - 1 with the pseudo-point
        p = Plan(spec, m=m, dtype="f32")
        n_quad = sum("a^2" in x for x in mods)
        assert p.alpha == m + 2 + n_quad                        # each quadratic adds one domain row
        assert p.tile_in + 0 <= p.alpha <= p.tile_in + 3        # a compiled (tile, alpha') pair
        p.close()


def test_candidate_count_and_order():
    sets = S.candidate_sets(4, max_quadratic=2)
    # 1 all-linear set, then 5 with one quadratic, then C(5,2) = 10 with two
    assert len(sets) == 1 + 5 + 10
    assert sets[0] == "0,-1,1,-1/2,2,inf"
    assert all("a^2" not in x for x in sets[0].split(","))
    assert S.candidate_sets(4, max_quadratic=0) == [sets[0]]
    no_inf = S.candidate_sets(2, max_quadratic=0, with_inf=False)
    assert no_inf == ["0,-1,1,-1/2"]


def test_x1_candidates_match_section_3_1():
    """Section 3.1: linear points from the list 0, -1, 1, -1/2, 2, 1/2, -2,
    -1/4, 4 and the quadratics a^2 + 1, a^2 + a + 1, a^2 - a + 1; every tile
    from 2 to 8 (odd ones included) gives valid plans of compiled shapes."""
    assert S.LINEAR_POINTS[:9] == ("0", "-1", "1", "-1/2", "2", "1/2", "-2", "-1/4", "4")
    assert S.QUADRATICS_X1 == ("a^2+1", "a^2+a+1", "a^2-a+1")
    for m in range(2, 9):
        sets = S.candidate_sets(m, max_quadratic=1, quadratics=S.QUADRATICS_X1)
        assert len(sets) == 4
        for spec in sets:
            p = Plan(spec, m=m, dtype="f32")
            assert p.alpha == m + 2 + S.n_quadratics(spec)
            p.close()


def test_normal_restricted_to_unit_interval():
    """The X1 draw: standard normal values restricted to (-1, 1)."""
    import numpy as np
    from paper_1905_05233_amd import workloads as WL
    x, w = WL.draw_inputs(4, 16, 16, 8, 8, "normal_clip1", seed=0)
    for a in (x, w):
        assert np.all(np.abs(a) < 1)
        assert abs(float(np.mean(a))) < 0.02
        # the variance of N(0, 1) restricted to (-1, 1) is 1 - 2 phi(1) / (2 Phi(1) - 1) = 0.2911
        assert abs(float(np.var(a)) - 0.2911) < 0.01
