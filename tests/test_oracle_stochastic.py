"""Pins of the oracle's speculative-sampling tree verification (§2.1): chains
reduce to the textbook left-to-right rule written out independently here,
the emitted token is distributed as the target (Monte Carlo, the lossless
property the paper states), and degenerate draft distributions."""
import numpy as np

from oracle import entmtp_oracle as orc


def softmax(z, it=1.0):
    y = np.asarray(z, np.float64) * it
    e = np.exp(y - y.max())
    return e / e.sum()


def textbook_chain(tokens, z, q, ua, us, it=1.0):
    """§2.1 on a chain 0 -> 1 -> ... -> n: keep token i with probability
    min(1, p(t)/p_hat(t)) (p, p_hat at its parent), else draw from
    norm(max(0, p - p_hat)) and stop; after the last token draw from p."""
    n = len(tokens) - 1
    for i in range(1, n + 1):
        p, qh = softmax(z[i - 1], it), np.asarray(q[i - 1], np.float64)
        t = tokens[i]
        ratio = np.inf if qh[t] == 0 else p[t] / qh[t]
        if not ua[i] < min(1.0, ratio):
            res = np.maximum(p - qh, 0)
            return i - 1, int(np.searchsorted(np.cumsum(res), us[i - 1] * res.sum(), side="right"))
    p = softmax(z[n], it)
    return n, int(np.searchsorted(np.cumsum(p), us[n] * p.sum(), side="right"))


def test_chain_is_the_textbook_rule():
    g = np.random.default_rng(3)
    for trial in range(300):
        n, V = int(g.integers(1, 6)), int(g.integers(2, 7))
        parent = [-1] + list(range(n))
        z = g.normal(0, 1.5, (n + 1, V))
        q = np.array([softmax(g.normal(0, 1.5, V)) for _ in range(n + 1)])
        tok = [0] + [int(g.integers(0, V)) for _ in range(n)]
        ua, us = g.random(n + 1), g.random(n + 1)
        a, path, bonus, best, _ = orc.accept_stochastic(parent, tok, z, q, 1.0, ua, us)
        ra, rbonus = textbook_chain(tok, z, q, ua, us)
        assert (a, bonus) == (ra, rbonus), trial
        assert path == list(range(a + 1))


def test_emitted_token_follows_the_target():
    """One node with two children drafted independently from q: the first
    emitted token (the accepted child's, or the residual draw) has the
    target's distribution p."""
    g = np.random.default_rng(11)
    V, N = 4, 40000
    z = np.array([[0.3, -0.2, 1.1, 0.0]] + [[0.0] * V] * 2)
    p = softmax(z[0])
    q = np.array([[0.1, 0.5, 0.15, 0.25]] + [[0.25] * V] * 2)
    counts = np.zeros(V)
    for _ in range(N):
        tok = [0] + [int(x) for x in g.choice(V, 2, p=q[0])]
        a, path, bonus, best, _ = orc.accept_stochastic([-1, 0, 0], tok, z, q, 1.0, g.random(3),
                                                        g.random(3))
        counts[tok[best] if a == 1 else bonus] += 1
    freq = counts / N
    assert np.all(np.abs(freq - p) < 5 * np.sqrt(p * (1 - p) / N)), (freq, p)


def test_draft_equal_to_target_accepts_first_children():
    g = np.random.default_rng(5)
    parent = [-1, 0, 0, 1, 1, 3, 2]
    V = 6
    z = g.normal(0, 1, (7, V))
    q = np.array([softmax(r) for r in z])
    tok = [0] + [int(g.integers(0, V)) for _ in range(6)]
    a, path, bonus, best, _ = orc.accept_stochastic(parent, tok, z, q, 1.0, g.random(7) * 0.999,
                                                    g.random(7))
    assert path == [0, 1, 3, 5] and a == 3       # r = q at the draft token: always kept


def test_impossible_draft_is_rejected_and_the_residual_is_the_target():
    # the draft token has target probability 0 (logit -inf): rejected for any
    # u, and max(0, p - q) = p, so the replacement is drawn from p itself
    z = np.array([[0.0, 0.0, -np.inf], [0.0, 0.0, 0.0]])
    q = np.array([[0.0, 0.0, 1.0], [1 / 3] * 3])
    for ua in (0.0, 0.5, 0.999):
        for us in (0.2, 0.7):
            a, path, bonus, best, _ = orc.accept_stochastic([-1, 0], [0, 2], z, q, 1.0, [0, ua],
                                                            [us, 0])
            assert a == 0 and bonus == (0 if us < 0.5 else 1)


def test_temperature_and_inverse_cdf_hand_example():
    # p at inv_temp 2 of logits ln[1, 2, 1] is [1, 4, 1] / 6: u = 0.5 -> cumsum 1/6, 5/6 -> index 1
    z = np.log(np.array([[1.0, 2.0, 1.0]]))
    a, path, bonus, best, _ = orc.accept_stochastic([-1], [0], z, np.ones((1, 3)) / 3, 2.0, [0], [0.5])
    assert (a, bonus) == (0, 1)
    a, path, bonus, best, _ = orc.accept_stochastic([-1], [0], z, np.ones((1, 3)) / 3, 2.0, [0], [0.9])
    assert bonus == 2
