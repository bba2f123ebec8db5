"""GPU parity of speculative-sampling tree verification (§2.1) against the
oracle, on seeded inputs whose every decision -- each acceptance test the
walk meets and the final draw -- stays clear of its threshold (fp32 on the
GPU, fp64 in the oracle, so both take the same decisions)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import entmtp_oracle as orc  # noqa: E402
from paper_2606_27550_amd import synth  # noqa: E402
from tests.helpers import dev_i32  # noqa: E402

pytestmark = pytest.mark.gpu

MARGIN_REL, MARGIN_ABS, DRAW_MARGIN = 1e-3, 1e-6, 1e-4


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


def say(*a):
    print("[gpu-test]", *a, flush=True)


def softmax(y):
    e = np.exp(y - y.max())
    return e / e.sum()


def make_inputs(g, parent, V, inv_temp, draft_from_target=False):
    """Peaked target logits (a few lifted tokens per row), draft
    distributions close to the target's, draft tokens drawn from the parent's
    draft distribution, and uniforms redrawn until every decision is clear."""
    T = len(parent)
    z = g.normal(0, 1, (T, V)).astype(np.float32)
    lift = np.log(V)   # lifts above the tail's total mass, so draws land on lifted tokens
    for i in range(T):
        z[i, g.integers(0, V, 6)] += (lift + g.uniform(-1, 3, 6)).astype(np.float32)
    if draft_from_target:
        q = np.array([softmax(z[i].astype(np.float64) * inv_temp) for i in range(T)], np.float32)
    else:
        q = np.array([softmax((z[i] + g.normal(0, 0.7, V)).astype(np.float64) * inv_temp)
                      for i in range(T)], np.float32)
    q64 = q.astype(np.float64)
    q64 /= q64.sum(axis=1, keepdims=True)
    tok = np.zeros(T, np.int64)
    for i in range(1, T):
        tok[i] = g.choice(V, p=q64[parent[i]])
    ua, us = g.random(T).astype(np.float32), g.random(T).astype(np.float32)
    for _ in range(200):
        res = orc.accept_stochastic(parent, tok, z.astype(np.float64), q.astype(np.float64),
                                    inv_temp, ua.astype(np.float64), us.astype(np.float64))
        bad = False
        for entry in res[4]:
            if entry[0] == "sample":
                _, tgt, lo, hi = entry
                if min(tgt - lo, hi - tgt) <= DRAW_MARGIN:
                    us[res[3]] = g.random()
                    bad = True
            else:
                c, lhs, rhs = entry
                if abs(lhs - rhs) <= MARGIN_REL * max(lhs, rhs) + MARGIN_ABS:
                    ua[c] = g.random()
                    bad = True
        if not bad:
            return z, q, tok, ua, us, res
    raise RuntimeError("no clear decisions")


def run(api, parent, z, q, tok, ua, us, inv_temp):
    """The statistics come from the library's own kernel at the same
    temperature, as they would in a verification step."""
    bank = api.Bank([parent])
    T, V = z.shape
    f = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()   # noqa: E731
    zd = f(z)
    H, p1 = torch.empty(T, device="cuda"), torch.empty(T, device="cuda")
    am = torch.empty(T, dtype=torch.int32, device="cuda")
    api.logit_stats(zd, inv_temp, H, p1, am)
    a = torch.full((1,), -3, dtype=torch.int32, device="cuda")
    path = torch.full((bank.D[0] + 1,), -9, dtype=torch.int32, device="cuda")
    bonus = torch.full((1,), -3, dtype=torch.int32, device="cuda")
    ws = torch.empty(V, dtype=torch.float32, device="cuda")
    api.accept_stochastic(bank, 0, dev_i32(tok), zd, f(q), inv_temp, am, p1, f(ua), f(us), ws, a,
                          path, bonus)
    torch.cuda.synchronize()
    return int(a.item()), path.cpu().numpy().tolist(), int(bonus.item())


@pytest.mark.parametrize("T,depth,V,inv_temp,seed", [(9, 3, 300, 1.0, 0), (26, 4, 4000, 1 / 0.7, 1),
                                                     (64, 5, 32000, 1.0, 2), (27, 4, 32000, 1 / 0.7, 3),
                                                     (8, 3, 128256, 1.0, 4)])
def test_stochastic_acceptance_matches_oracle(api, T, depth, V, inv_temp, seed):
    g = np.random.default_rng(100 + seed)
    parent = synth.uniform_attach_tree(90 + seed, T, depth)
    for rep in range(6):
        z, q, tok, ua, us, ref = make_inputs(g, parent, V, inv_temp)
        ra, rpath, rbonus, rbest, trace = ref
        say(f"stochastic T {T} V {V} rep {rep}: oracle accept {ra}, {len(trace) - 1} tests, "
            f"bonus {rbonus}")
        a, path, bonus = run(api, parent, z, q, tok, ua, us, inv_temp)
        assert (a, bonus) == (ra, rbonus)
        assert path[: a + 1] == list(rpath) and all(x == -1 for x in path[a + 1:])


def test_chain_and_draft_equal_to_target(api):
    g = np.random.default_rng(7)
    chain = list(range(-1, 5))
    for rep in range(4):
        z, q, tok, ua, us, ref = make_inputs(g, chain, 1000, 1.0)
        assert run(api, chain, z, q, tok, ua, us, 1.0)[::2] == (ref[0], ref[2])
    # q = p: the first child of every accepted node passes
    parent = [-1, 0, 0, 1, 1, 3, 2]
    z, q, tok, ua, us, ref = make_inputs(g, parent, 500, 1.0, draft_from_target=True)
    a, path, bonus = run(api, parent, z, q, tok, ua, us, 1.0)
    assert path[: a + 1] == [0, 1, 3, 5] == list(ref[1]) and bonus == ref[2]


def test_invalid_draft_token_is_rejected(api):
    """A draft token outside the vocabulary never passes, and the residual
    update follows as for any rejection: the same walk as the oracle's with a
    token the root's test clearly rejects in its place."""
    g = np.random.default_rng(8)
    parent = [-1, 0, 0, 1]
    checked = 0
    for rep in range(8):
        z, q, tok, ua, us, _ = make_inputs(g, parent, 200, 1.0)
        p0 = softmax(z[0].astype(np.float64))
        t_rej = int(np.argmax(q[0].astype(np.float64) / p0))   # q(t) well above p(t)
        if q[0][t_rej] <= 1.05 * p0[t_rej]:   # (u = 0.999 then rejects it clearly)
            continue
        ua_ref = ua.astype(np.float64)
        ua_ref[1] = 0.999
        tok_ref = tok.copy()
        tok_ref[1] = t_rej
        ref = orc.accept_stochastic(parent, tok_ref, z.astype(np.float64), q.astype(np.float64),
                                    1.0, ua_ref, us.astype(np.float64))
        clear = all(e[0] == "sample" or abs(e[1] - e[2]) > MARGIN_REL * max(e[1], e[2]) + MARGIN_ABS
                    for e in ref[4]) and min(ref[4][-1][1] - ref[4][-1][2],
                                             ref[4][-1][3] - ref[4][-1][1]) > DRAW_MARGIN
        if not clear:
            continue
        tok_bad = tok.copy()
        tok_bad[1] = 10 ** 6
        a, path, bonus = run(api, parent, z, q, tok_bad, ua, us, 1.0)
        assert (a, bonus) == (ref[0], ref[2]) and path[: a + 1] == list(ref[1])
        checked += 1
    assert checked >= 3
