"""The paper's data-movement model (oracle.cost_model) against its pins (CPU only).

Pins: the R_A worked example and the counts the paper states (golden file),
the matmul closed form Eq. (3), Eq. (5) and the seven other closed forms of
Sec. 4, the compulsory volume at T = N, and a brute-force simulation of an
ideal cache that keeps exactly the previous tile (the model's assumption in
Sec. 2.2 / 3.1), which counts moved elements by explicit index sets.
"""
import itertools
import json
import math
import os
import random
from fractions import Fraction

import pytest

from oracle import cost_model as cm

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_model_facts.json")))


def divisors(n):
    return [d for d in range(1, n + 1) if n % d == 0]


def rand_problem(rng, hi=12):
    N = {j: rng.choice([x for x in range(1, hi + 1)]) for j in cm.ITERS}
    T = {j: rng.choice(divisors(N[j])) for j in cm.ITERS}
    return N, T


# ---------------------------------------------------------------- golden facts

def test_counts_stated_in_paper():
    assert math.factorial(7) == GOLD["tile_loop_permutations_one_level"]["value"]
    assert len(cm.CLASSES) == GOLD["pruned_classes"]["value"]
    three = math.factorial(7) ** 3
    assert abs(three - GOLD["three_level_configurations"]["value"]) / three < 0.01
    four = math.factorial(7) ** 4
    assert abs(four - GOLD["four_level_cases"]["value"]) / four < 0.01


def test_class_sizes_and_disjointness():
    sizes = [len(cm.class_members(ci)) for ci in range(8)]
    assert sizes[:4] == [GOLD["class_members_4_2_bands"]["value"]] * 4
    assert sizes[4:] == [120] * 4  # 5! orders of the outer band
    seen = set()
    for ci in range(8):
        for p in cm.class_members(ci):
            assert p not in seen
            seen.add(p)
    for ci, rep in enumerate(cm.REPRESENTATIVES):
        assert cm.class_of(rep) == ci


def test_r_a_worked_example():
    ex = GOLD["r_a_example"]
    rest = [x for x in cm.ITERS if x not in ex["perm_suffix"]]
    for head in itertools.permutations(rest):
        p = tuple(head) + tuple(ex["perm_suffix"])
        assert cm.r_position("Out", p) == ex["R_Out"]
        assert cm.r_position("In", p) == ex["R_In"]
        assert cm.r_position("Ker", p) == ex["R_Ker"]


# ---------------------------------------------------------------- closed forms

def test_matmul_eq3():
    """Unit h, w, r, s extents turn Eq. (1) into a matmul (i=n, j=k, k=c);
    with the reduction tile loop innermost the volume is Eq. (3)."""
    rng = random.Random(3)
    for _ in range(200):
        Ni, Nj, Nk = rng.randint(1, 40), rng.randint(1, 40), rng.randint(1, 40)
        Ti, Tj, Tk = rng.choice(divisors(Ni)), rng.choice(divisors(Nj)), rng.choice(divisors(Nk))
        N = dict(n=Ni, k=Nj, c=Nk, r=1, s=1, h=1, w=1)
        T = dict(n=Ti, k=Tj, c=Tk, r=1, s=1, h=1, w=1)
        eq3 = Ni * Nj * Nk * (Fraction(1, Tj) + Fraction(1, Ti) + Fraction(2, Nk))
        for unit_order in itertools.permutations("rshw"):
            p = tuple(unit_order) + ("n", "k", "c")
            assert cm.data_volume(p, N, T) == eq3


def _r(N, T, j):
    return Fraction(N[j], T[j])


def closed_form(ci, N, T):
    """The paper's printed expression for class ``ci`` (Sec. 4: Eq. (5) and the
    expressions after it).  Readings: the In footprint printed with T_k for the
    innermost-s and innermost-r classes is read with T_n (In has no k index);
    the full seven-ratio forms are used for the innermost-k classes."""
    r = lambda j: _r(N, T, j)  # noqa: E731
    Tn, Tk, Tc, Tr, Ts, Th, Tw = (T[j] for j in "nkcrshw")
    out = Tn * Tk * Th * Tw
    ker = Tk * Tc * Tr * Ts
    allr = r("n") * r("k") * r("c") * r("r") * r("s") * r("h") * r("w")
    if ci == 0:  # Eq. (5)
        return r("k") * r("c") * r("r") * r("s") * (
            ker + r("n") * r("h") * (2 * r("w") * out + Tn * Tc * (Th + Tr - 1) * (N["w"] + Ts - 1)))
    if ci == 1:
        return r("k") * r("c") * r("r") * r("s") * (
            ker + r("n") * r("w") * (2 * r("h") * out + Tn * Tc * (Tw + Ts - 1) * (N["h"] + Tr - 1)))
    if ci in (2, 3):
        dv_out = 2 * r("n") * r("k") * r("h") * r("w") * out
        dv_ker = allr * ker
        if ci == 2:
            dv_in = r("n") * r("k") * r("c") * r("r") * r("w") * r("h") * Tn * Tc * (Th + Tr - 1) * (Tw + N["s"] - 1)
        else:
            dv_in = r("n") * r("k") * r("c") * r("s") * r("w") * r("h") * Tn * Tc * (Th + N["r"] - 1) * (Tw + Ts - 1)
        return dv_out + dv_ker + dv_in
    dv_out = 2 * allr * out
    dv_ker = allr * ker
    if ci == 4:
        dv_in = r("n") * r("c") * r("r") * r("s") * r("h") * Tn * Tc * (Th + Tr - 1) * (N["w"] + Ts - 1)
    elif ci == 5:
        dv_in = r("n") * r("c") * r("r") * r("s") * r("w") * Tn * Tc * (N["h"] + Tr - 1) * (Tw + Ts - 1)
    elif ci == 6:
        dv_in = r("n") * r("c") * r("r") * r("h") * r("w") * Tn * Tc * (Th + Tr - 1) * (Tw + N["s"] - 1)
    else:
        dv_in = r("n") * r("c") * r("s") * r("h") * r("w") * Tn * Tc * (Th + N["r"] - 1) * (Tw + Ts - 1)
    return dv_out + dv_ker + dv_in


@pytest.mark.parametrize("ci", range(8))
def test_class_closed_forms(ci):
    rng = random.Random(100 + ci)
    for _ in range(300):
        N, T = rand_problem(rng)
        assert cm.data_volume(cm.REPRESENTATIVES[ci], N, T) == closed_form(ci, N, T)


def test_full_tiles_give_compulsory_volume():
    rng = random.Random(5)
    for _ in range(50):
        N, _ = rand_problem(rng)
        comp = (N["n"] * N["c"] * (N["h"] + N["r"] - 1) * (N["w"] + N["s"] - 1)
                + N["k"] * N["c"] * N["r"] * N["s"] + 2 * N["n"] * N["k"] * N["h"] * N["w"])
        for p in rng.sample(list(itertools.permutations(cm.ITERS)), 40):
            assert cm.data_volume(p, N, dict(N)) == comp


# ---------------------------------------------------------------- pruning

def test_class_members_share_one_cost():
    rng = random.Random(7)
    members = [cm.class_members(ci) for ci in range(8)]
    for _ in range(6):
        N, T = rand_problem(rng)
        for ci in range(8):
            vals = {cm.data_volume(p, N, T) for p in members[ci]}
            assert len(vals) == 1, (ci, N, T)


def test_pruning_to_eight_classes_is_lossless():
    """Sec. 4's claim, checked pointwise in T: for every tile vector the best of
    the eight representatives is as good as the best of all 5040 orders."""
    rng = random.Random(9)
    allp = list(itertools.permutations(cm.ITERS))
    for _ in range(8):
        N, T = rand_problem(rng, hi=16)
        best_all = min(cm.data_volume(p, N, T) for p in allp)
        best_rep = min(cm.data_volume(p, N, T) for p in cm.REPRESENTATIVES)
        assert best_rep == best_all, (N, T)


# ---------------------------------------------------------------- brute force

def _tile_sets(o, T):
    """Index sets each array touches in the tile at origin ``o`` (enumerated)."""
    rn = range(o["n"], o["n"] + T["n"])
    rk = range(o["k"], o["k"] + T["k"])
    rc = range(o["c"], o["c"] + T["c"])
    rr = range(o["r"], o["r"] + T["r"])
    rs = range(o["s"], o["s"] + T["s"])
    rh = range(o["h"], o["h"] + T["h"])
    rw = range(o["w"], o["w"] + T["w"])
    out = set(itertools.product(rn, rk, rh, rw))
    ker = set(itertools.product(rk, rc, rr, rs))
    inp = {(n, c, h + r, w + s) for n in rn for c in rc for h in rh for r in rr for w in rw for s in rs}
    return {"In": inp, "Ker": ker, "Out": out}


def simulate_previous_tile_cache(perm, N, T):
    """Elements loaded per array when the cache holds exactly the previous
    tile's data: sum over tiles of |footprint(t) minus footprint(t-1)|."""
    ranges = [range(N[j] // T[j]) for j in perm]
    prev = {a: set() for a in cm.ARRAYS}
    vol = {a: 0 for a in cm.ARRAYS}
    for iv in itertools.product(*ranges):
        o = {j: iv[i] * T[j] for i, j in enumerate(perm)}
        cur = _tile_sets(o, T)
        for a in cm.ARRAYS:
            vol[a] += len(cur[a] - prev[a])
        prev = cur
    return vol


PAIR = {"w": "s", "s": "w", "h": "r", "r": "h"}


def test_rule_matches_previous_tile_cache_simulation():
    """Where the model's assumption holds exactly -- every present iterator
    really changes on a wrap (N_j/T_j >= 2), and a wrapped sliding window does
    not overlap the previous one (N_x >= 2 T_x + 2 T_y - 1 for the sliding
    pair (x, y) at R_In) -- the rule of Sec. 3.2 equals the simulation."""
    rng = random.Random(11)
    allp = list(itertools.permutations(cm.ITERS))
    compared = 0
    cases = 0
    while cases < 10:
        T = {j: rng.choice([1, 1, 2]) for j in cm.ITERS}
        N = {j: T[j] * rng.choice([2, 3]) for j in cm.ITERS}
        for x in "wshr":
            N[x] = T[x] * max(2, -(-(2 * T[x] + 2 * T[PAIR[x]] - 1) // T[x]))
        if math.prod(N[j] // T[j] for j in cm.ITERS) > 1500:
            continue
        cases += 1
        for p in rng.sample(allp, 12):
            sim = simulate_previous_tile_cache(p, N, T)
            for a in cm.ARRAYS:
                assert cm.array_volume(a, p, N, T) == sim[a], (a, p, N, T)
            compared += 1
    assert compared >= 100


# ---------------------------------------------------------------- multi-level

def test_multilevel_reduces_to_single_level():
    rng = random.Random(13)
    for _ in range(30):
        N, T0 = rand_problem(rng)
        p0, p1 = rng.sample(list(itertools.permutations(cm.ITERS)), 2)
        dv = cm.level_volumes([p0, p1], [T0, dict(N)], N)
        assert dv[0] == cm.data_volume(p0, N, T0)
        assert dv[1] == cm.data_volume(p1, N, N)
        assert cm.level_volumes([p0], [T0], N) == [cm.data_volume(p0, N, T0)]


def test_multilevel_counts_outer_tiles():
    """With the level-1 tile a 1/m-th slice of N along one iterator, level 0 is
    the single-level model of that slice, repeated m times."""
    rng = random.Random(17)
    for _ in range(30):
        N, T0 = rand_problem(rng)
        j = rng.choice([x for x in cm.ITERS if N[x] // T0[x] >= 2 and (N[x] // T0[x]) % 2 == 0] or ["n"])
        if (N[j] // T0[j]) % 2:
            continue
        T1 = dict(N)
        T1[j] = N[j] // 2
        p0 = rng.choice(list(itertools.permutations(cm.ITERS)))
        dv = cm.level_volumes([p0, cm.REPRESENTATIVES[0]], [T0, T1], N)
        assert dv[0] == 2 * cm.data_volume(p0, T1, T0)


def test_minmax_objective_hand_computed():
    """Sec. 5 objective on a two-level example worked by hand, with the
    dominant level switching with the bandwidths.

    N = (n1 k2 c2 r1 s1 h1 w4); level-0 tile T0 = (n1 k1 c1 r1 s1 h1 w4) in
    the order n,k,h,w,c,r,s; level 1 is the whole problem.
    Level 0 (Sec. 3.2 rule, positions counted from the innermost s = 1):
      In  -- innermost present iterator s (sliding case, N_s - T_s = 0):
             (N/T over n,k,h,w,c,r = 1*2*1*1*2*1 = 4) x footprint 1*1*1*4 = 16
      Ker -- innermost present s: ratio over all seven = 4, footprint 1 -> 4
      Out -- innermost present w (position 4): ratio over n,k,h,w = 2,
             footprint 4 -> 8, read and written -> 16
      DV^0 = 36.
    Level 1 (T = N): compulsory In 8 + Ker 4 + 2 * Out 8 = 28.
    """
    N = dict(n=1, k=2, c=2, r=1, s=1, h=1, w=4)
    T0 = dict(n=1, k=1, c=1, r=1, s=1, h=1, w=4)
    perms = [cm.REPRESENTATIVES[2], cm.REPRESENTATIVES[0]]
    assert cm.level_volumes(perms, [T0, dict(N)], N) == [36, 28]
    # DV^0 / 4 = 9 < DV^1 / 1 = 28: level 1 bounds
    assert cm.minmax_cost(perms, [T0, dict(N)], N, [4, 1]) == 28
    # DV^0 / 1 = 36 > DV^1 / 4 = 7: level 0 bounds
    assert cm.minmax_cost(perms, [T0, dict(N)], N, [1, 4]) == 36
    # equal bandwidths of 3: max(12, 28/3) = 12
    assert cm.minmax_cost(perms, [T0, dict(N)], N, [3, 3]) == 12


def test_capacity_eq4_hand_computed():
    """Eq. (4) on a tile worked by hand: T = (n1 k4 c2 r3 s3 h3 w6) touches
    In 1*2*(3+3-1)*(6+3-1) = 80, Ker 4*2*3*3 = 72 and Out 1*4*3*6 = 72
    elements, 224 in all."""
    T = dict(n=1, k=4, c=2, r=3, s=3, h=3, w=6)
    assert [cm.footprint(a, T) for a in cm.ARRAYS] == [80, 72, 72]
    assert cm.capacity_ok(T, 224)
    assert not cm.capacity_ok(T, 223)


def test_footprints_count_distinct_elements_brute_force():
    """Each footprint of Sec. 3.1 equals the number of distinct elements one
    tile touches, enumerated index by index from Eq. (1)'s subscripts."""
    rng = random.Random(29)
    for _ in range(40):
        T = {j: rng.randint(1, 4) for j in cm.ITERS}
        o = {j: rng.randint(0, 5) for j in cm.ITERS}  # tile origin
        rng_ = {j: range(o[j], o[j] + T[j]) for j in cm.ITERS}
        ins, kers, outs = set(), set(), set()
        for n in rng_["n"]:
            for k in rng_["k"]:
                for c in rng_["c"]:
                    for r in rng_["r"]:
                        for s_ in rng_["s"]:
                            for h in rng_["h"]:
                                for w in rng_["w"]:
                                    ins.add((n, c, h + r, w + s_))
                                    kers.add((k, c, r, s_))
                                    outs.add((n, k, h, w))
        assert cm.footprint("In", T) == len(ins)
        assert cm.footprint("Ker", T) == len(kers)
        assert cm.footprint("Out", T) == len(outs)
        total = len(ins) + len(kers) + len(outs)
        assert cm.capacity_ok(T, total) and not cm.capacity_ok(T, total - 1)
