"""Oracle for the paper's analytical data-movement model -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the smoke check and the benchmark's cpu_baseline leg may import
this module; the product's tile selector is a separate C++ implementation that
shares no code with it.

Everything is computed in exact rational arithmetic (``fractions.Fraction``) so
that a comparison with another implementation can be bit-exact.

Notation (Sec. 3): the seven loop iterators are n, k, c, r, s, h, w.  ``N`` and
``T`` map each iterator to its problem extent and tile size.  As in Listing 2,
the h and w extents are the *output* extents (the input index is h + r).  A
permutation is a tuple of iterators from outermost to innermost, i.e. the
paper's <i7, ..., i1>; the position of an iterator is 1 for the innermost.

Functions and the passages they follow:

* ``footprint``            -- tile footprints, Sec. 3.1 (the terms of Eq. (4)).
* ``capacity_ok``          -- capacity constraint, Eq. (4).
* ``r_position``           -- R_A, Sec. 3.1 (innermost present iterator).
* ``array_volume``         -- the two-case cost rule of Sec. 3.2.
* ``data_volume``          -- sum over In, Ker, Out; Out counted twice (read
                              and write, Sec. 2.2 and Sec. 4 "Innermost wt").
* ``CLASSES`` / ``class_of`` / ``class_members`` -- the eight permutation
                              classes of the summary of Sec. 4.
* ``multilevel_volumes``   -- Sec. 5: level-l volume with problem extents
                              replaced by the next outer tile sizes.
* ``minmax_cost``          -- the objective of Sec. 5, max over levels of
                              DV^l / BW^l.
"""
from fractions import Fraction
from itertools import permutations
from math import prod

ITERS = ("n", "k", "c", "r", "s", "h", "w")

# Which loop iterators index each tensor (Sec. 4: each iterator is present in
# exactly two of the three tensors).
PRESENT = {
    "In": frozenset("nchrws"),
    "Ker": frozenset("kcrs"),
    "Out": frozenset("nkhw"),
}

ARRAYS = ("In", "Ker", "Out")

# Iterators for which In has partial (sliding) reuse between consecutive
# tiles: its index expressions are h + r and w + s (Sec. 3.2, second case).
SLIDING = frozenset("whsr")


def _chk(N, T):
    for j in ITERS:
        if not (1 <= T[j] <= N[j]):
            raise ValueError(f"tile size T[{j}]={T[j]} outside 1..N[{j}]={N[j]}")


def footprint(array, T):
    """Elements of ``array`` touched by one tile (Sec. 3.1)."""
    if array == "In":
        return T["n"] * T["c"] * (T["h"] + T["r"] - 1) * (T["w"] + T["s"] - 1)
    if array == "Ker":
        return T["k"] * T["c"] * T["r"] * T["s"]
    if array == "Out":
        return T["n"] * T["k"] * T["h"] * T["w"]
    raise KeyError(array)


def capacity_ok(T, capacity):
    """Eq. (4): the three footprints of one tile fit in ``capacity`` words."""
    return sum(footprint(a, T) for a in ARRAYS) <= capacity


def positions(perm):
    """Position of each iterator in ``perm`` (outer->inner), innermost = 1."""
    if sorted(perm) != sorted(ITERS):
        raise ValueError(f"not a permutation of the seven iterators: {perm}")
    L = len(perm)
    return {x: L - i for i, x in enumerate(perm)}


def r_position(array, perm):
    """R_A: innermost position of an iterator present in ``array``."""
    pos = positions(perm)
    return min(pos[x] for x in PRESENT[array])


def array_volume(array, perm, N, T):
    """Data moved for one array over the whole tiled execution (Sec. 3.2).

    Case 1 (Out, Ker, and In when the iterator at R_In is n or c): every
    change of the iterator at R_A (or of any outer iterator) brings a disjoint
    slice, so the volume is the footprint times the product of N_j/T_j over
    the positions R_A..7.

    Case 2 (In when the iterator at R_In is w, h, s or r): consecutive tiles
    along that iterator overlap, so only the non-overlapping part moves.  The
    volume is the product of N_j/T_j over the positions strictly outside R_In,
    times (full footprint for the first tile + the new data for the remaining
    N_x/T_x - 1 steps, which replaces one extent of the footprint by N_x - T_x).
    """
    _chk(N, T)
    pos = positions(perm)
    ra = r_position(array, perm)
    it_at_ra = perm[len(perm) - ra]
    if array == "In" and it_at_ra in SLIDING:
        outer = prod((Fraction(N[j], T[j]) for j in ITERS if pos[j] > ra), start=Fraction(1))
        base = T["n"] * T["c"]
        hh = T["h"] + T["r"] - 1
        ww = T["w"] + T["s"] - 1
        if it_at_ra == "w":
            partial = base * hh * (N["w"] - T["w"])
        elif it_at_ra == "s":
            partial = base * hh * (N["s"] - T["s"])
        elif it_at_ra == "h":
            partial = base * (N["h"] - T["h"]) * ww
        else:  # "r"
            partial = base * (N["r"] - T["r"]) * ww
        return outer * (footprint("In", T) + partial)
    ratio = prod((Fraction(N[j], T[j]) for j in ITERS if pos[j] >= ra), start=Fraction(1))
    return ratio * footprint(array, T)


def data_volume(perm, N, T, out_factor=2):
    """Total modelled volume DV = DV_In + DV_Ker + out_factor * DV_Out.

    ``out_factor`` is 2 in the paper (each Out element is read and written).
    """
    return (array_volume("In", perm, N, T) + array_volume("Ker", perm, N, T)
            + out_factor * array_volume("Out", perm, N, T))


def volumes(perm, N, T, out_factor=2):
    """Per-array volumes as a dict (Out already multiplied by out_factor)."""
    return {
        "In": array_volume("In", perm, N, T),
        "Ker": array_volume("Ker", perm, N, T),
        "Out": out_factor * array_volume("Out", perm, N, T),
    }


# ---------------------------------------------------------------------------
# The eight permutation classes (summary of Sec. 4).  Each class is a sequence
# of bands from outermost to innermost; the order inside a band is free.
CLASSES = (
    (frozenset("kcrs"), frozenset("nh"), frozenset("w")),
    (frozenset("kcrs"), frozenset("nw"), frozenset("h")),
    (frozenset("nkhw"), frozenset("cr"), frozenset("s")),
    (frozenset("nkhw"), frozenset("cs"), frozenset("r")),
    (frozenset("nchrs"), frozenset("w"), frozenset("k")),
    (frozenset("ncwrs"), frozenset("h"), frozenset("k")),
    (frozenset("nchwr"), frozenset("s"), frozenset("k")),
    (frozenset("nchws"), frozenset("r"), frozenset("k")),
)

# One fixed representative per class (outer -> inner).  The first two are the
# examples the paper itself gives for the innermost-w and innermost-h classes.
REPRESENTATIVES = (
    ("k", "c", "r", "s", "n", "h", "w"),
    ("k", "c", "r", "s", "n", "w", "h"),
    ("n", "k", "h", "w", "c", "r", "s"),
    ("n", "k", "h", "w", "c", "s", "r"),
    ("n", "c", "h", "r", "s", "w", "k"),
    ("n", "c", "w", "r", "s", "h", "k"),
    ("n", "c", "h", "w", "r", "s", "k"),
    ("n", "c", "h", "w", "s", "r", "k"),
)


def class_of(perm):
    """Index 0..7 of the class containing ``perm``, or None."""
    for ci, bands in enumerate(CLASSES):
        i = 0
        ok = True
        for band in bands:
            if frozenset(perm[i:i + len(band)]) != band:
                ok = False
                break
            i += len(band)
        if ok:
            return ci
    return None


def class_members(ci):
    return [p for p in permutations(ITERS) if class_of(p) == ci]


# ---------------------------------------------------------------------------
# Multi-level tiling (Sec. 5).

def level_volumes(perms, tiles, N, out_factor=2):
    """Modelled volume DV^l at each level l = 0 (innermost) .. L-1.

    ``tiles[l]`` is the level-l tile; the level above level L-1 is the whole
    problem.  Within one level-(l+1) tile the level-l tile loops run over the
    ranges T^{l+1}_j (Sec. 5), so the single-level rule applies with N
    replaced by T^{l+1}; the whole execution runs prod_j N_j / T^{l+1}_j such
    level-(l+1) tiles.
    """
    L = len(tiles)
    if len(perms) != L:
        raise ValueError("one permutation per level")
    out = []
    for l in range(L):
        upper = tiles[l + 1] if l + 1 < L else N
        for j in ITERS:
            if tiles[l][j] > upper[j]:
                raise ValueError(f"level {l} tile exceeds the level above in {j}")
        reps = prod((Fraction(N[j], upper[j]) for j in ITERS), start=Fraction(1))
        out.append(reps * data_volume(perms[l], upper, tiles[l], out_factor))
    return out


def minmax_cost(perms, tiles, N, bandwidths, out_factor=2):
    """Sec. 5 objective: max over levels of DV^l / BW^l."""
    dv = level_volumes(perms, tiles, N, out_factor)
    return max(Fraction(d) / Fraction(bw) for d, bw in zip(dv, bandwidths))
