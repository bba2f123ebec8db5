"""Pins of the oracle's typical acceptance (not the GPU): degenerate
thresholds, closed forms for uniform logits, equivalence with greedy
acceptance on peaked distributions, hand-worked examples, and the choice
among equally deep accepted nodes checked by brute force."""
import math

import numpy as np

from oracle import entmtp_oracle as orc
from paper_2606_27550_amd import synth


def tree_and_tokens(seed, T=27, depth=4, V=10):
    g = np.random.default_rng(seed)
    parent = synth.uniform_attach_tree(seed, T, depth)
    return parent, g.integers(0, V, T), g


def test_zero_threshold_accepts_the_whole_tree():
    parent, tok, g = tree_and_tokens(1)
    z = g.standard_normal((len(parent), 10))
    a, path, _, best, p, thr = orc.accept_typical(parent, tok, z, 1 / 0.7, 0.0, 0.3)
    assert a == synth.tree_depth(parent)
    assert (thr == 0.0).all() and (p[1:] > 0).all()


def test_uniform_logits_closed_form():
    V = 10
    parent, tok, _ = tree_and_tokens(2, V=V)
    z = np.zeros((len(parent), V))
    # p = 1/V everywhere, H = ln V, threshold = min(eps, alpha / V)
    a, *_ = orc.accept_typical(parent, tok, z, 1.0, 0.09, 0.3)        # 0.03 < 0.1: accept
    assert a == synth.tree_depth(parent)
    a, *_ = orc.accept_typical(parent, tok, z, 1.0, 0.5, 2.0)         # min(0.5, 0.2) > 0.1
    assert a == 0
    a, *_ = orc.accept_typical(parent, tok, z, 1.0, 0.09, 2.0)        # min(0.09, 0.2) < 0.1
    assert a == synth.tree_depth(parent)
    _, _, _, _, p, thr = orc.accept_typical(parent, tok, z, 1.0, 0.5, 2.0)
    assert np.allclose(thr, 0.2) and np.allclose(p[1:], 0.1)


def test_peaked_distributions_reduce_to_greedy():
    for seed in range(5):
        V = 50
        parent, _, g = tree_and_tokens(10 + seed, V=V)
        T = len(parent)
        am = g.integers(0, V, T)
        z = np.zeros((T, V))
        z[np.arange(T), am] = 1000.0          # one token holds all the mass: H = 0
        tok = synth.draft_tokens(parent, am, g.random(T), g.integers(0, V, T), 0.7)
        ra, rpath, rbonus, rbest = orc.accept(parent, tok, am)
        a, path, bonus, best, _, thr = orc.accept_typical(parent, tok, z, 1 / 0.7, 0.09, 0.3)
        assert (a, list(path), bonus, best) == (ra, list(rpath), rbonus, rbest)
        assert np.allclose(thr, 0.09)


def test_hand_worked_three_token_example():
    # parent distribution p = (0.6, 0.3, 0.1) from logits (ln 6, ln 3, ln 1)
    parent = [-1, 0, 0, 0]
    z = np.array([[math.log(6), math.log(3), 0.0]] + [[0.0, 0.0, 0.0]] * 3)
    tok = [0, 0, 1, 2]
    H = -(0.6 * math.log(0.6) + 0.3 * math.log(0.3) + 0.1 * math.log(0.1))   # 0.8979 nats
    assert abs(0.3 * math.exp(-H) - 0.12222) < 1e-4
    # eps 0.09: threshold 0.09, every child (0.6, 0.3, 0.1) passes
    a, path, bonus, best, p, thr = orc.accept_typical(parent, tok, z, 1.0, 0.09, 0.3)
    assert np.allclose(p[1:], [0.6, 0.3, 0.1]) and abs(thr[0] - 0.09) < 1e-12
    assert (a, best) == (1, 1) and bonus == 0            # the most likely depth-1 node (0.6)
    # the same children with their tokens permuted: the 0.6 child is node 2
    a, path, _, best, p, _ = orc.accept_typical(parent, [0, 2, 0, 1], z, 1.0, 0.09, 0.3)
    assert np.allclose(p[1:], [0.1, 0.6, 0.3]) and (a, best, list(path)) == (1, 2, [0, 2])
    # equal tokens are equally likely: the lowest index wins
    a, _, _, best, _, _ = orc.accept_typical(parent, [0, 1, 1, 2], z, 1.0, 0.09, 0.3)
    assert (a, best) == (1, 1)
    # eps 0.2: threshold 0.3 * exp(-H) = 0.1222; the 0.1 child fails, 0.3 passes
    a, _, _, _, _, thr = orc.accept_typical(parent, [0, 2, 2, 1], z, 1.0, 0.2, 0.3)
    assert abs(thr[0] - 0.3 * math.exp(-H)) < 1e-12 and a == 1
    a, *_ = orc.accept_typical(parent, [0, 2, 2, 2], z, 1.0, 0.2, 0.3)
    assert a == 0
    # temperature 0.5 sharpens to (36, 9, 1) / 46: the 9/46 = 0.196 child passes
    # min(0.2, 0.3 exp(-H')) only because H' is smaller
    p2 = np.array([36, 9, 1]) / 46
    H2 = -(p2 * np.log(p2)).sum()
    _, _, _, _, p, thr = orc.accept_typical(parent, [0, 1, 1, 1], z, 2.0, 0.2, 0.3)
    assert np.allclose(p[1:], 9 / 46) and abs(thr[0] - min(0.2, 0.3 * math.exp(-H2))) < 1e-12


def test_threshold_is_the_parents_and_strict():
    # parent (0.6, 0.3, 0.1): threshold min(0.5, 0.45 exp(-H)) = 0.183; the
    # child row is peaked (H = 0): its own threshold would be min(0.5, 0.45)
    parent = [-1, 0]
    z = np.array([[math.log(6), math.log(3), 0.0], [1000.0, 0.0, 0.0]])
    a, _, _, _, _, thr = orc.accept_typical(parent, [0, 1], z, 1.0, 0.5, 0.45)   # 0.3 > 0.183
    assert a == 1 and abs(thr[0] - 0.45 * 0.40740) < 1e-4 and thr[1] == 0.45
    # p exactly equal to the threshold is not enough: uniform V = 10 gives
    # p = 1/10, and eps = 0.1 with a large alpha makes the threshold 0.1
    z = np.zeros((2, 10))
    a, _, _, _, p, thr = orc.accept_typical(parent, [0, 3], z, 1.0, 0.1, 5.0)
    assert p[1] == 0.1 and thr[0] == 0.1 and a == 0


def test_deepest_tie_goes_to_the_most_likely_path():
    # parent = [-1, 0, 0, 1, 2]: nodes 1, 2 at depth 1, node 3 under 1, node 4 under 2.
    # root p = (0.6, 0.3, 0.1); node 1 p = (0.7, 0.2, 0.1); node 2 p = (0.4, 0.35, 0.25)
    parent = [-1, 0, 0, 1, 2]
    z = np.log(np.array([[0.6, 0.3, 0.1], [0.7, 0.2, 0.1], [0.4, 0.35, 0.25],
                         [1 / 3, 1 / 3, 1 / 3], [1 / 3, 1 / 3, 1 / 3]]))
    # node 1 drafts token 1 (0.3), node 2 token 0 (0.6); node 3 token 0 under
    # node 1 (0.7), node 4 token 0 under node 2 (0.4).  Both depth-2 nodes pass
    # (threshold <= 0.09); their paths: 0.3 * 0.7 = 0.21 < 0.6 * 0.4 = 0.24, so
    # node 4 is chosen although its own token is the less likely one
    a, path, bonus, best, p, _ = orc.accept_typical(parent, [0, 1, 0, 0, 0], z, 1.0, 0.09, 0.3)
    assert np.allclose(p[1:], [0.3, 0.6, 0.7, 0.4])
    assert (a, best, list(path), bonus) == (2, 4, [0, 2, 4], 0)
    # node 3's token made 0.9 likely: 0.27 > 0.24, node 3 wins
    z[1] = np.log([0.9, 0.05, 0.05])
    a, path, _, best, _, _ = orc.accept_typical(parent, [0, 1, 0, 0, 0], z, 1.0, 0.09, 0.3)
    assert (a, best, list(path)) == (2, 3, [0, 1, 3])


def test_choice_among_deepest_matches_brute_force():
    """The chosen node maximises the product of its path's draft
    probabilities (computed here as a product, not as a sum of logs) over
    every accepted node of the greatest depth, lowest index on ties."""
    V = 6
    for seed in range(40):
        g = np.random.default_rng(300 + seed)
        T = int(g.integers(2, 30))
        parent = synth.uniform_attach_tree(300 + seed, T, int(g.integers(1, min(5, T))))
        z = g.standard_normal((T, V)) * 0.3         # flat rows: many siblings pass together
        tok = g.integers(0, V, T)
        a, path, _, best, p, thr = orc.accept_typical(parent, tok, z, 1.0, 0.09, 0.3)
        acc = [True] + [False] * (T - 1)
        for i in range(1, T):
            acc[i] = acc[parent[i]] and p[i] > thr[parent[i]]
        depth = [0] * T
        for i in range(1, T):
            depth[i] = depth[parent[i]] + 1
        top = max(depth[i] for i in range(T) if acc[i])
        def prob(i):
            out = 1.0
            while i != 0:
                out *= p[i]
                i = parent[i]
            return out
        cands = [i for i in range(T) if acc[i] and depth[i] == top]
        want = min(cands, key=lambda i: (-prob(i), i))
        assert (a, best) == (top, want), (seed, cands)
        assert list(path) == orc.ancestors_or_self(parent, want)
