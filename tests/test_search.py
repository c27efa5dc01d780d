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
