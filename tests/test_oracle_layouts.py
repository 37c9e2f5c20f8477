"""Pins for candidate layout lists and the view predicate."""
import itertools
import math

import numpy as np
import pytest

from oracle import brute, layouts


def test_layout_list_counts_and_identity_first():
    assert len(layouts.layout_list((3, 4, 5))) == 6
    assert len(layouts.layout_list((2, 3, 4, 5))) == 24
    # extent-1 dims do not create new physical orders
    assert len(layouts.layout_list((1, 4, 5))) == 2
    assert len(layouts.layout_list((1, 12, 128, 64))) == 6
    assert len(layouts.layout_list((1, 1, 7))) == 1
    for s in [(3, 4, 5), (1, 4, 5), (2, 1, 3, 1)]:
        lst = layouts.layout_list(s)
        assert lst[0] == tuple(range(len(s)))
        assert lst == sorted(lst)                      # lexicographic
        keys = [layouts.physical_key(s, p) for p in lst]
        assert len(set(keys)) == len(keys)
        r = len(s)
        nontriv = [d for d in s if d != 1]
        assert len(lst) == math.factorial(len(nontriv))


def test_strides_match_numpy_transpose():
    rng = np.random.default_rng(0)
    shape = (2, 3, 4, 5)
    x = rng.standard_normal(shape)
    for p in itertools.permutations(range(4)):
        st = layouts.strides(shape, p)
        phys = np.ascontiguousarray(x.transpose(p)).ravel()
        for _ in range(10):
            i = tuple(int(rng.integers(0, s)) for s in shape)
            assert phys[sum(a * b for a, b in zip(i, st))] == x[i]


CASES = [
    ("transpose", (0, 2, 1, 3), (1, 4, 2, 3), (1, 2, 4, 3)),
    ("transpose", (0, 2, 3, 1), (2, 4, 2, 3), (2, 2, 3, 4)),
    ("transpose", (1, 0, 2), (3, 1, 4), (1, 3, 4)),
    ("reshape", None, (1, 4, 6), (1, 4, 2, 3)),
    ("reshape", None, (2, 4, 6), (2, 4, 2, 3)),
    ("reshape", None, (2, 4, 2, 3), (2, 4, 6)),
    ("reshape", None, (3, 1, 6), (3, 1, 2, 3)),
    ("reshape", None, (2, 6), (2, 1, 6)),
]


@pytest.mark.parametrize("op,perm,xs,ys", CASES)
def test_view_predicate_equals_offset_definition(op, perm, xs, ys):
    for lin in itertools.permutations(range(len(xs))):
        for lout in itertools.permutations(range(len(ys))):
            want = brute.view_by_offsets(op, perm, xs, ys, lin, lout)
            got = layouts.is_view(op, perm, xs, ys, lin, lout)
            assert got == want, (lin, lout)


def test_identity_layouts_make_reshapes_views_and_transposes_copies():
    assert layouts.is_view("reshape", None, (2, 4, 6), (2, 4, 2, 3), (0, 1, 2), (0, 1, 2, 3))
    assert not layouts.is_view("transpose", (0, 2, 1, 3), (2, 4, 2, 3), (2, 2, 4, 3),
                               (0, 1, 2, 3), (0, 1, 2, 3))
    # a transposed input layout makes the transpose a view
    assert layouts.is_view("transpose", (0, 2, 1, 3), (2, 4, 2, 3), (2, 2, 4, 3),
                           (0, 1, 2, 3), (0, 2, 1, 3))
