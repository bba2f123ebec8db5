"""GPU parity of typical acceptance (draft-token logits + the typical
acceptance walk) against the oracle, on inputs whose every draft token's
probability stays at least 1% away from its threshold (so fp32 and fp64 take
the same decisions), and on peaked rows where it must equal greedy."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import entmtp_oracle as orc  # noqa: E402
from paper_2606_27550_amd import synth  # noqa: E402
from tests.helpers import dev_bf16, dev_i32, margin_hidden  # noqa: E402

pytestmark = pytest.mark.gpu

INV_T, EPS, ALPHA = 1 / 0.7, 0.09, 0.3


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


def say(*a):
    print("[gpu-test]", *a, flush=True)


def separated_drafts(parent, z, am, g, V):
    """Drafts mixing argmax tokens, top-k tokens and random tokens, each kept
    only when its probability is >= 1% away from the parent's threshold."""
    T = len(parent)
    probs, thr = [], []
    for j in range(T):
        p, H = orc.typical_probs(z[j], INV_T)
        probs.append(p)
        thr.append(min(EPS, ALPHA * np.exp(-H)))
    tok = np.zeros(T, np.int64)
    for i in range(1, T):
        pj, tj = probs[parent[i]], thr[parent[i]]
        order = np.argsort(-pj)
        for _ in range(200):
            kind = g.random()
            t = am[parent[i]] if kind < 0.5 else (order[g.integers(0, 5)] if kind < 0.8 else g.integers(0, V))
            if abs(pj[t] - tj) > 0.01 * tj:
                tok[i] = t
                break
        else:
            raise RuntimeError("no separated draft")
    return tok


def deepest_loglik(parent, p, thr):
    """The accepted nodes of the greatest depth and the fp64 log-likelihood
    of each one's path (the quantity the tie-break compares)."""
    T = len(parent)
    acc, depth, ll = [True] + [False] * (T - 1), [0] * T, [0.0] * T
    for i in range(1, T):
        depth[i] = depth[parent[i]] + 1
        acc[i] = acc[parent[i]] and p[i] > thr[parent[i]]
        if acc[i]:
            ll[i] = ll[parent[i]] + np.log(p[i])
    top = max(depth[i] for i in range(T) if acc[i])
    return [(i, ll[i]) for i in range(T) if acc[i] and depth[i] == top]


def tie_separated(parent, tok, p, thr, gap=1e-3):
    """fp32 and fp64 choose the same node among the deepest: the winner's
    path log-likelihood leads every other by `gap`, or the runners-up are
    exact copies of it (the same draft tokens along the same parents)."""
    c = sorted(deepest_loglik(parent, p, thr), key=lambda x: -x[1])
    if len(c) < 2:
        return True
    best = c[0]
    for i, l in c[1:]:
        if best[1] - l >= gap:
            continue
        same = tok[i] == tok[best[0]] and parent[i] == parent[best[0]]
        if not same:
            return False
    return True


def run_typical(api, parent, X, W, tok):
    T, hid = X.shape
    V = W.shape[0]
    bank = api.Bank([parent])
    Xd, Wd = dev_bf16(X), dev_bf16(W)
    logits = torch.empty((T, V), device="cuda")
    H, p1 = torch.empty(T, device="cuda"), torch.empty(T, device="cuda")
    am = torch.empty(T, dtype=torch.int32, device="cuda")
    ws = torch.empty(api.verify_logits_stats_workspace(T, hid, V), dtype=torch.uint8, device="cuda")
    api.verify_logits_stats(Xd, Wd, logits, INV_T, H, p1, am, ws)
    zd, zt = torch.empty(T, device="cuda"), torch.empty(T, device="cuda")
    tok_d = dev_i32(tok)
    api.draft_logits(bank, 0, Xd, Wd, tok_d, am, zd, zt)
    a = torch.zeros(1, dtype=torch.int32, device="cuda")
    path = torch.full((bank.D[0] + 1,), -7, dtype=torch.int32, device="cuda")
    bonus = torch.zeros(1, dtype=torch.int32, device="cuda")
    best = torch.zeros(1, device="cuda")
    api.accept_typical(bank, 0, tok_d, am, zd, zt, H, p1, INV_T, EPS, ALPHA, a, path, bonus, best)
    torch.cuda.synchronize()
    return (int(a.item()), path.cpu().numpy(), int(bonus.item()), float(best.item()),
            zd.cpu().numpy(), zt.cpu().numpy(), p1.cpu().numpy())


@pytest.mark.parametrize("T,depth,hid,V,spike", [(27, 4, 512, 1000, False), (64, 5, 1024, 4000, True),
                                                 (128, 6, 4096, 32000, True), (9, 3, 256, 300, False)])
def test_typical_acceptance_matches_oracle(api, T, depth, hid, V, spike):
    say("typical acceptance", T, hid, V)
    g = np.random.default_rng(T + V)
    parent = synth.uniform_attach_tree(40 + T, T, depth)
    W = synth.lm_head_weight(40 + T, V, hid, std=0.05)
    if spike:   # confident rows (the regime typical acceptance is built for)
        deltas = g.uniform(4.0, 12.0)
        X = margin_hidden(40 + T, T, W, spikes=(deltas, g.integers(0, V, T)), w_std=0.05)
    else:
        X = margin_hidden(40 + T, T, W)
    z = orc.verify_logits(X, W).astype(np.float32).astype(np.float64)
    am = z.argmax(axis=1)
    for _ in range(50):
        tok = separated_drafts(parent, z, am, g, V)
        ra, rpath, rbonus, rbest, rp, rthr = orc.accept_typical(parent, tok, z, INV_T, EPS, ALPHA)
        if tie_separated(parent, tok, rp, rthr):
            break
    else:
        raise RuntimeError("no draft set with a separated choice among the deepest nodes")
    local = rp[1:] > rthr[np.asarray(parent[1:])]
    beyond_greedy = sum(1 for i in range(1, T) if local[i - 1] and tok[i] != am[parent[i]])
    assert 0 < local.sum() < T - 1 or T < 16
    assert beyond_greedy > 0       # the case differs from greedy acceptance
    a, path, bonus, best, zd, zt, p1 = run_typical(api, parent, X, W, tok)
    say(f"  accept {a} (oracle {ra}); nodes accepted locally {int(local.sum())} of {T - 1}, "
        f"{beyond_greedy} of them not the argmax")
    assert (a, bonus) == (ra, rbonus)
    assert path[: a + 1].tolist() == list(rpath)
    assert (path[a + 1:] == -1).all()
    assert abs(best - p1[rbest]) == 0.0
    # the draft logits themselves: X[parent] . W[tok] in fp32
    Xf, Wf = orc.bf16_to_f64(X), orc.bf16_to_f64(W)
    for i in range(1, T):
        assert abs(zd[i] - Xf[parent[i]] @ Wf[tok[i]]) <= 1e-4 * max(1.0, abs(z).max())
        assert abs(zt[i] - Xf[parent[i]] @ Wf[am[parent[i]]]) <= 1e-4 * max(1.0, abs(z).max())


@pytest.mark.parametrize("T,depth,hid,V", [(27, 4, 512, 1000), (64, 5, 1024, 4000), (128, 6, 4096, 32000)])
def test_typical_chooses_the_most_likely_deepest_path(api, T, depth, hid, V):
    """Flat rows (small hidden states): nearly every draft passes, many nodes
    share the greatest depth, and the choice among them is the path whose
    drafts are jointly most likely, not the lowest index."""
    say("typical tie-break", T, hid, V)
    g = np.random.default_rng(7 * T + V)
    parent = synth.uniform_attach_tree(70 + T, T, depth)
    W = synth.lm_head_weight(70 + T, V, hid, std=0.05)
    X = margin_hidden(70 + T, T, W)
    z = orc.verify_logits(X, W).astype(np.float32).astype(np.float64)
    am = z.argmax(axis=1)
    for _ in range(50):
        tok = separated_drafts(parent, z, am, g, V)
        ra, rpath, rbonus, rbest, rp, rthr = orc.accept_typical(parent, tok, z, INV_T, EPS, ALPHA)
        cands = deepest_loglik(parent, rp, rthr)
        if len(cands) > 1 and rbest != cands[0][0] and tie_separated(parent, tok, rp, rthr):
            break
    else:
        raise RuntimeError("no draft set whose deepest tie the likelihood decides")
    a, path, bonus, best, *_ = run_typical(api, parent, X, W, tok)
    say(f"  accept {a} (oracle {ra}), chosen {rbest} among {[c for c, _ in cands]}")
    assert (a, bonus) == (ra, rbonus)
    assert path[: a + 1].tolist() == list(rpath)
    assert (path[a + 1:] == -1).all()


def test_typical_equals_greedy_on_peaked_rows(api):
    """Rows whose top logit leads by a wide margin: every non-argmax draft is
    far below the threshold and every argmax draft far above it."""
    T, hid, V = 27, 512, 1000
    g = np.random.default_rng(5)
    parent = synth.uniform_attach_tree(55, T, 4)
    W = synth.lm_head_weight(55, V, hid, std=0.05)
    am0 = g.integers(0, V, T)
    X = synth.plant_spike(synth.hidden_rows(55, T, hid), W, am0, 40.0, 0.05)
    z = orc.verify_logits(X, W).astype(np.float32).astype(np.float64)
    am = z.argmax(axis=1)
    tok = synth.draft_tokens(parent, am, g.random(T), g.integers(0, V, T), 0.7)
    ra, rpath, rbonus, _ = orc.accept(parent, tok, am)
    a, path, bonus, *_ = run_typical(api, parent, X, W, tok)
    assert (a, bonus) == (ra, rbonus) and path[: a + 1].tolist() == list(rpath)


def test_out_of_range_draft_is_rejected(api):
    T, hid, V = 5, 256, 100
    parent = [-1, 0, 1, 2, 3]
    W = synth.lm_head_weight(66, V, hid, std=0.05)
    X = synth.hidden_rows(66, T, hid)
    z = orc.verify_logits(X, W).astype(np.float32)
    am = z.argmax(axis=1)
    tok = np.array([0, am[0], V + 7, am[2], am[3]])    # node 2 carries an invalid token
    a, path, bonus, best, zd, zt, p1 = run_typical(api, parent, X, W, tok)
    assert zd[2] == -np.inf and a == 1
