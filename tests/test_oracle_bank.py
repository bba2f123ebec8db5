"""Pins of the oracle's TopologyBank buffers (tree mask, position offsets,
gather / retrieve indices; §2.3 and §4 "Cost").

Pinned by: a hand-worked fixture, brute force over every tree with up to 7
nodes against the transitive closure of the parent relation (Warshall), and
structural invariants (chain, star, popcount = depth + 1).
"""
import itertools

import numpy as np
import pytest

from oracle import entmtp_oracle as orc
from tests.conftest import golden


def all_parent_arrays(T):
    """Every parent array with parent[i] in [0, i)."""
    for tail in itertools.product(*[range(i) for i in range(1, T)]):
        yield [-1] + list(tail)


def warshall_closure(parent):
    T = len(parent)
    R = np.eye(T, dtype=bool)
    for i in range(1, T):
        R[i, parent[i]] = True          # i reaches its parent
    for k in range(T):
        R = R | (R[:, [k]] & R[[k], :])
    return R                              # R[i, j]: j is i or an ancestor of i


def mask_bits(mask_row, T):
    return np.array([(int(mask_row[j // 32]) >> (j % 32)) & 1 for j in range(orc.T_MAX)], dtype=bool)


def test_hand_worked_tree():
    g = golden("tree7_buffers.json")
    e = orc.bank_entry(g["parent"])
    assert e["depth"].tolist() == g["depth"]
    assert e["mask"][:, 0].tolist() == g["mask_word0"]
    assert (e["mask"][:, 1:] == 0).all()
    assert e["path"].tolist() == g["path"]
    assert e["leaves"].tolist() == g["leaves"]
    assert e["retrieve"].tolist() == g["retrieve"]


@pytest.mark.parametrize("T", range(1, 8))
def test_bruteforce_masks_against_closure(T):
    n = 0
    for parent in all_parent_arrays(T):
        e = orc.bank_entry(parent)
        R = warshall_closure(parent)
        for i in range(T):
            bits = mask_bits(e["mask"][i], T)
            assert (bits[:T] == R[i]).all()
            assert not bits[T:].any()
            assert e["depth"][i] == R[i].sum() - 1          # popcount = depth + 1
            # the path row lists exactly the closure, ordered by depth
            p = e["path"][i]
            chain = p[p >= 0]
            assert sorted(chain.tolist()) == np.flatnonzero(R[i]).tolist()
            assert chain[-1] == i and chain[0] == 0
            assert len(chain) == e["depth"][i] + 1
        n += 1
    assert n == max(1, int(np.prod(range(1, T))))


def test_chain_is_lower_triangular_and_star_is_diag_plus_root():
    T = 32
    e = orc.bank_entry([-1] + list(range(T - 1)))
    for i in range(T):
        assert mask_bits(e["mask"][i], T)[:T].tolist() == [j <= i for j in range(T)]
    assert e["leaves"].tolist() == [T - 1]
    e = orc.bank_entry([-1] + [0] * (T - 1))
    for i in range(T):
        assert mask_bits(e["mask"][i], T)[:T].tolist() == [j == 0 or j == i for j in range(T)]
    assert e["leaves"].tolist() == list(range(1, T))


def test_mask_recursion_on_random_trees():
    rng = np.random.default_rng(0)
    for T in (2, 33, 100, 256):
        parent = [-1] + [int(rng.integers(i)) for i in range(1, T)]
        try:
            e = orc.bank_entry(parent)
        except ValueError:
            continue                                          # deeper than D_MAX
        for i in range(1, T):
            expect = e["mask"][parent[i]].copy()
            expect[i // 32] |= np.uint32(1 << (i % 32))
            assert (e["mask"][i] == expect).all()


@pytest.mark.parametrize("parent", [[], [0], [-1, 1], [-1, 0, 2], [-1, 0, -1], [-1] * 2])
def test_invalid_trees_rejected(parent):
    with pytest.raises(ValueError):
        orc.bank_entry(parent)


def test_size_and_depth_limits():
    with pytest.raises(ValueError):
        orc.bank_entry([-1] + [0] * orc.T_MAX)               # T_MAX + 1 nodes
    orc.bank_entry([-1] + [0] * (orc.T_MAX - 1))             # exactly T_MAX
    orc.bank_entry([-1] + list(range(orc.D_MAX)))            # depth D_MAX
    with pytest.raises(ValueError):
        orc.bank_entry([-1] + list(range(orc.D_MAX + 1)))    # depth D_MAX + 1
