"""Pins of the oracle's greedy tree acceptance (§2.1 left-to-right acceptance,
greedy case; accept length of §5.1), KV compaction (§3.2 decode loop) and the
hysteretic ladder scheduler (§4 Policy).

Independent references: hand-worked fixtures, brute force over every
root-to-node path of every tree with up to 6 nodes, the per-leaf cumulative
product rule used by Medusa-style verifiers, and the special cases the method
has (all drafts match, none match, one node, chain mismatches).
"""
import itertools

import numpy as np
import pytest

from oracle import entmtp_oracle as orc
from paper_2606_27550_amd import synth
from tests.conftest import golden
from tests.test_oracle_bank import all_parent_arrays


def test_hand_worked_accept_and_compaction():
    g = golden("tree7_accept.json")
    for case in g["cases"]:
        a, path, bonus, best = orc.accept(g["parent"], case["draft"], g["target_argmax"])
        assert (a, path, bonus) == (case["accept_len"], case["path"], case["bonus"])
        assert best == path[-1]
    c = g["compaction"]
    rows = np.array(c["rows_before"], dtype=np.uint16)
    k = np.repeat(rows[None, :, None], 2, axis=0).repeat(3, axis=2)   # [H=2, cap, d=3]
    k2, v2 = orc.kv_compact(k, k + 100, c["prefix_len"], c["path"])
    assert k2[0, :, 0].tolist() == c["rows_after"]
    assert (v2[1, :, 2] - 100).tolist() == c["rows_after"]


def bruteforce_accept(parent, tok, am):
    """Enumerate every root-to-node path; a path is accepted when every edge's
    child token equals the parent's greedy token; keep the longest, first in
    node order."""
    T = len(parent)
    best = (0, [0])
    for node in range(T):
        chain = orc.ancestors_or_self(parent, node)
        if all(tok[c] == am[p] for p, c in zip(chain, chain[1:])):
            if len(chain) - 1 > best[0]:
                best = (len(chain) - 1, chain)
    return best


def test_bruteforce_small_trees():
    g = np.random.default_rng(0)
    for T in range(1, 7):
        for parent in all_parent_arrays(T):
            for _ in range(6):
                am = g.integers(0, 3, T)
                tok = g.integers(0, 3, T)
                a, path, bonus, _ = orc.accept(parent, tok, am)
                ra, rpath = bruteforce_accept(parent, tok, am)
                assert (a, path) == (ra, rpath)
                assert bonus == am[path[-1]]


def test_special_cases():
    g = np.random.default_rng(1)
    for n, cap in ((27, 4), (64, 5), (128, 6)):
        parent = synth.uniform_attach_tree(1, n, cap)
        am = g.integers(0, 32000, n)
        all_match = np.array([-1] + [am[parent[i]] for i in range(1, n)])
        a, path, bonus, best = orc.accept(parent, all_match, am)
        assert a == cap == synth.tree_depth(parent)
        none = all_match.copy()
        none[1:] += 1
        a, path, bonus, best = orc.accept(parent, none, am)
        assert (a, path, bonus) == (0, [0], am[0])
    a, path, bonus, _ = orc.accept([-1], [-1], [42])
    assert (a, path, bonus) == (0, [0], 42)
    # chain with its first mismatch at depth k accepts k - 1 drafts
    T = 9
    parent = synth.chain_tree(T)
    am = np.arange(100, 100 + T)
    for k in range(1, T):
        tok = np.array([-1] + [am[i - 1] for i in range(1, T)])
        tok[k] = 7
        assert orc.accept(parent, tok, am)[0] == k - 1


def medusa_leaf_rule(entry, tok, am):
    """Per-candidate rule: for each root-to-leaf row, the accept length is the
    number of leading matches (cumulative product of matches); the candidate
    with the largest count wins (first in leaf order)."""
    best_len, best_leaf = -1, -1
    for l, row in enumerate(entry["retrieve"]):
        row = row[row >= 0]
        m = np.cumprod([tok[c] == am[p] for p, c in zip(row, row[1:])] or [1])
        n = int(m.sum()) if len(row) > 1 else 0
        if n > best_len:
            best_len, best_leaf = n, l
    return best_len, entry["retrieve"][best_leaf][: best_len + 1].tolist()


def test_equivalence_with_per_leaf_cumprod_rule():
    g = np.random.default_rng(2)
    for trial in range(300):
        n = int(g.integers(2, 40))
        parent = synth.uniform_attach_tree(50 + trial, n, int(g.integers(1, min(n - 1, 6) + 1)))
        entry = orc.bank_entry(parent)
        am = g.integers(0, 4, n)
        tok = np.array([-1] + [am[parent[i]] if g.random() < 0.7 else g.integers(0, 4)
                               for i in range(1, n)])
        a, path, _, _ = orc.accept(parent, tok, am)
        la, lpath = medusa_leaf_rule(entry, tok, am)
        assert a == la
        # sibling tokens all distinct -> the accepted set is a single chain
        children = {}
        for i in range(1, n):
            children.setdefault(parent[i], []).append(int(tok[i]))
        if all(len(v) == len(set(v)) for v in children.values()):
            assert path == lpath


def test_compaction_identity_and_bruteforce():
    g = np.random.default_rng(4)
    k = g.integers(0, 65535, (3, 4, 40, 8)).astype(np.uint16)     # [layers, H, cap, d]
    v = g.integers(0, 65535, (3, 4, 40, 8)).astype(np.uint16)
    k2, v2 = orc.kv_compact(k, v, 20, [0, 1, 2, 3])
    np.testing.assert_array_equal(k2, k)
    np.testing.assert_array_equal(v2, v)
    path = [0, 2, 5, 6, 11]
    k2, v2 = orc.kv_compact(k, v, 20, path)
    for row in range(40):
        if 20 <= row < 25:
            src = 20 + path[row - 20]
        else:
            src = row
        np.testing.assert_array_equal(k2[:, :, row], k[:, :, src])
        np.testing.assert_array_equal(v2[:, :, row], v[:, :, src])


def test_ladder_hand_trace():
    g = golden("ladder_trace.json")
    rung = 0
    for s, want in zip(g["s"], g["rungs"]):
        rung = orc.ladder_next(rung, g["n_rungs"], s, g["tau_on"], g["tau_off"])
        assert rung == want
    big = False
    for s, want in ((0.81, True), (0.7, True), (0.6, False), (0.7, False), (0.8, False), (0.9, True)):
        big = orc.binary_next(big, s, 0.8, 0.6)
        assert big == want
