"""Pins of the oracle's Algorithm 1 scoring step (§3.1): the frontier of a
tree, one-node augmentations scored from one rollout of the joint tree
(checked against scoring every augmented tree on its own with the greedy
acceptance oracle), and the tie-broken choice of the node to add."""
import numpy as np

from oracle import entmtp_oracle as orc


def tuples(parent):
    """Each node's Medusa-style name: its child ranks from the root."""
    rank = orc.child_ranks(parent)
    return [tuple(rank[j] for j in orc.ancestors_or_self(parent, i)[1:]) for i in range(len(parent))]


def test_next_children_hand_example():
    # T = {(0)}: the root proposes (1), node (0) proposes (0, 0)
    joint, in_tree = orc.joint_tree([-1, 0], 2)
    assert tuples(joint) == [(), (0,), (1,), (0, 0)]
    assert in_tree == [True, True, False, False]
    # depth 1 is the limit: only the root may grow
    assert orc.joint_tree([-1, 0], 1)[0] == [-1, 0, 0]
    # a chain of depth 2 with D = 2: the deepest node proposes nothing
    assert tuples(orc.joint_tree([-1, 0, 1], 2)[0]) == [(), (0,), (0, 0), (1,), (0, 1)]
    assert orc.rank_sums([-1, 0, 1, 0, 1]) == [0, 0, 0, 1, 1]


def test_hand_worked_scores_and_choice():
    # T = chain (0), (0, 0); D = 3 -> candidates (1), (0, 1), (0, 0, 0)
    joint, in_tree = orc.joint_tree([-1, 0, 1], 3)
    assert tuples(joint) == [(), (0,), (0, 0), (1,), (0, 1), (0, 0, 0)]
    ok = [[1, 1, 1, 0, 1, 1],      # T accepts to depth 2; (0,1) accepted at 2, (0,0,0) at 3
          [1, 0, 1, 1, 1, 1]]      # (0) fails: T gives 0; only (1) is accepted, at depth 1
    sums = orc.frontier_scores(joint, in_tree, ok)
    assert sums == [2, 2, 2, 3, 2, 3]
    # (1) and (0,0,0) tie at 3: the smaller rank sum (0 < 1) wins, though deeper
    assert orc.frontier_select(joint, in_tree, sums) == 5


def test_tie_breaks_rank_sum_then_depth_then_index():
    joint, in_tree = orc.joint_tree([-1, 0, 1], 3)   # candidates 3: (1), 4: (0,1), 5: (0,0,0)
    # (1) and (0,1) both have rank sum 1; with equal scores the shallower wins
    assert orc.frontier_select(joint, in_tree, [0, 0, 0, 7, 7, 6]) == 3
    # a higher score beats every tie-break
    assert orc.frontier_select(joint, in_tree, [0, 0, 0, 6, 7, 6]) == 4
    # all equal: rank sum 0 wins
    assert orc.frontier_select(joint, in_tree, [0, 0, 0, 5, 5, 5]) == 5
    # identical keys: the lower index (two candidates under the same parent
    # cannot share a rank, so this needs a hand-made in_tree)
    assert orc.frontier_select([-1, 0, 0], [True, False, False], [0, 3, 3]) == 1
    assert orc.frontier_select([-1, 0], [True, True], [1, 1]) == -1   # no candidate


def test_scores_equal_scoring_each_augmented_tree_alone():
    """The single rollout of T u F gives, for every candidate, what greedy
    acceptance on T u {nu} alone gives, summed over the samples."""
    g = np.random.default_rng(31)
    for trial in range(60):
        n = int(g.integers(1, 12))
        parent = [-1] + [int(g.integers(0, i)) for i in range(1, n)]
        D = max(orc.depths(parent)) + int(g.integers(0, 3))
        D = max(D, 1)
        joint, in_tree = orc.joint_tree(parent, D)
        J = len(joint)
        S = 25
        V = int(g.integers(2, 5))            # few tokens: frequent matches
        tok = g.integers(0, V, (S, J))
        am = g.integers(0, V, (S, J))
        ok = [[i == 0 or tok[s][i] == am[s][joint[i]] for i in range(J)] for s in range(S)]
        sums = orc.frontier_scores(joint, in_tree, ok)
        members = [i for i in range(J) if in_tree[i]]
        for i in range(J):
            keep = members if in_tree[i] else members + [i]
            remap = {old: new for new, old in enumerate(keep)}
            sub = [-1] + [remap[joint[k]] for k in keep[1:]]
            total = 0
            for s in range(S):
                a, *_ = orc.accept(sub, [int(tok[s][k]) for k in keep], [int(am[s][k]) for k in keep])
                total += a
            assert sums[i] == total, (trial, i)


def test_all_accepted_and_none_accepted():
    joint, in_tree = orc.joint_tree([-1, 0, 1, 0], 4)
    d = orc.depths(joint)
    dT = max(d[i] for i in range(len(joint)) if in_tree[i])
    ones = [[1] * len(joint)] * 3
    assert orc.frontier_scores(joint, in_tree, ones) == \
        [3 * (dT if in_tree[i] else max(dT, d[i])) for i in range(len(joint))]
    zeros = [[1] + [0] * (len(joint) - 1)] * 3
    assert orc.frontier_scores(joint, in_tree, zeros) == [0] * len(joint)
