"""GPU tests of the batched entry points whose per-sequence choices (tree
indices, prefix lengths, row offsets) live in device memory.

For the same trees, prefix lengths and rows they must give exactly what the
host-array batched calls give (the kernels derive the host's plan), so
outputs, cache appends, acceptance and compaction are compared bit for bit
with those calls, which the oracle pins (tests/test_gpu_batched.py); one case
is also checked against the oracle directly.  Entries the host cannot check
(a tree index outside the bank, a prefix that leaves no room for the tree, a
row range that is not the tree's) make that sequence do nothing.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import entmtp_oracle as orc  # noqa: E402
from paper_2606_27550_amd import synth  # noqa: E402
from tests.helpers import dev_bf16, dev_i32, host_bits  # noqa: E402

pytestmark = pytest.mark.gpu

ATOL_BF16 = 2e-2
WL = synth.WORKLOADS["batch8_gqa_v128k"]
D_HEAD = 128
THETA = 10000.0
SCALE = 1 / math.sqrt(D_HEAD)


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


@pytest.fixture(scope="module")
def trees():
    return synth.workload_trees(WL)


def say(*a):
    print("[gpu-test]", *a, flush=True)


def inputs(trees, topo, lens, Hq, Hkv, cap, seed):
    inp = [synth.attn_inputs(seed, len(trees[t]), Hq, Hkv, D_HEAD, L, cap, step=b + 1)
           for b, (t, L) in enumerate(zip(topo, lens))]
    return inp


def host_attn(api, bank, inp, topo, lens, Hq, Hkv):
    cat = lambda name: dev_bf16(np.ascontiguousarray(np.concatenate([getattr(x, name) for x in inp])))
    q, kt, vt = cat("q"), cat("k_tree"), cat("v_tree")
    kcs = [dev_bf16(x.k_cache) for x in inp]
    vcs = [dev_bf16(x.v_cache) for x in inp]
    out = torch.full((q.shape[0], Hq, D_HEAD), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(api.tree_attn_batched_workspace(len(topo), max(bank.T), Hq, Hkv, D_HEAD, max(lens)),
                     dtype=torch.uint8, device="cuda")
    api.tree_attn_batched(bank, topo, lens, q, kt, vt, kcs, vcs, SCALE, THETA, out, ws)
    torch.cuda.synchronize()
    return host_bits(out), [host_bits(k) for k in kcs], [host_bits(v) for v in vcs]


def device_attn(api, bank, inp, topo, lens, Hq, Hkv, cap, row_off, rows_cap, fill=7.0):
    """Rows of sequence b at row_off[b] in buffers of rows_cap rows (other
    rows of q / k_tree / v_tree zero, of out `fill`)."""
    B = len(topo)
    q = np.zeros((rows_cap, Hq, D_HEAD), np.uint16)
    kt = np.zeros((rows_cap, Hkv, D_HEAD), np.uint16)
    vt = np.zeros((rows_cap, Hkv, D_HEAD), np.uint16)
    for b in range(B):
        T = inp[b].q.shape[0]
        r0 = int(row_off[b])
        if 0 <= r0 and r0 + T <= rows_cap:
            q[r0:r0 + T], kt[r0:r0 + T], vt[r0:r0 + T] = inp[b].q, inp[b].k_tree, inp[b].v_tree
    kcs = [dev_bf16(x.k_cache) for x in inp]
    vcs = [dev_bf16(x.v_cache) for x in inp]
    out = torch.full((rows_cap, Hq, D_HEAD), fill, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(api.tree_attn_batched_device_workspace(bank, B, Hq, Hkv, D_HEAD, cap),
                     dtype=torch.uint8, device="cuda")
    api.tree_attn_batched_device(bank, dev_i32(np.asarray(topo, np.int32)),
                                 dev_i32(np.asarray(lens, np.int32)),
                                 dev_i32(np.asarray(row_off, np.int32)), dev_bf16(q), dev_bf16(kt),
                                 dev_bf16(vt), kcs, vcs, SCALE, THETA, out, ws)
    torch.cuda.synchronize()
    return host_bits(out), [host_bits(k) for k in kcs], [host_bits(v) for v in vcs]


@pytest.mark.parametrize("topo,lens,Hq,Hkv", [
    ([0, 4, 2, 1, 3, 4], [0, 37, 300, 513, 90, 1000], 8, 2),
    ([1, 2, 0, 3, 4, 2, 1, 0], [700, 64, 1500, 1023, 2048, 5, 129, 3000], WL.n_heads, WL.n_kv_heads),
    ([3], [777], 8, 8),                       # a batch of one (the lone-sequence split rule)
    ([0, 0, 1], [10, 2000, 31], 8, 2),        # small trees only: the one-tile instance
])
def test_attn_device_arrays_equal_host_arrays(api, trees, topo, lens, Hq, Hkv):
    say("tree_attn_batched_device", topo, lens, Hq, Hkv)
    bank = api.Bank(trees)
    cap = max(lens) + 128 + 5
    inp = inputs(trees, topo, lens, Hq, Hkv, cap, 301)
    h_out, h_k, h_v = host_attn(api, bank, inp, topo, lens, Hq, Hkv)
    Ts = [len(trees[t]) for t in topo]
    row_off = np.concatenate([[0], np.cumsum(Ts)]).astype(np.int32)
    d_out, d_k, d_v = device_attn(api, bank, inp, topo, lens, Hq, Hkv, cap, row_off, int(row_off[-1]))
    np.testing.assert_array_equal(d_out, h_out)
    for b in range(len(topo)):
        np.testing.assert_array_equal(d_k[b], h_k[b])
        np.testing.assert_array_equal(d_v[b], h_v[b])


def test_attn_device_arrays_rows_anywhere_and_invalid_entries(api, trees):
    """Sequences at gapped row offsets match the oracle; a tree index outside
    the bank, a prefix leaving no room for the tree and a row range shorter
    than the tree leave their output rows and caches untouched."""
    Hq, Hkv = 8, 2
    n = len(trees)
    cap = 1024
    topo = [2, n, 3, 1, 4, 4]
    Ts = [len(trees[t]) if t < n else 8 for t in topo]
    lens = [300, 50, cap - Ts[2] + 1, 900, 120, 10]      # sequence 2: one slot short
    bank = api.Bank(trees)
    inp = inputs(trees, [min(t, n - 1) for t in topo], [min(L, cap - 128) for L in lens], Hq, Hkv,
                 cap, 302)
    row_off = np.zeros(7, np.int32)
    row_off[0] = 5
    row_off[1] = row_off[0] + Ts[0] + 3                  # a gap of three rows
    row_off[2] = row_off[1] + 9
    row_off[3] = 200
    row_off[4] = row_off[3] + Ts[3] - 1                  # sequence 3: one row short
    rows_cap = int(row_off[4]) + Ts[4] + 6
    row_off[5] = 2**31 - 100                             # sequence 5: rows past 2^31
    row_off[6] = 2**31 - 1
    assert row_off[2] + Ts[2] <= row_off[3]
    d_out, d_k, d_v = device_attn(api, bank, inp, topo, lens, Hq, Hkv, cap, row_off, rows_cap)
    fill_bits = host_bits(torch.full((1,), 7.0, dtype=torch.bfloat16, device="cuda"))[0]
    done = np.zeros(rows_cap, bool)
    for b in (0, 4):
        t, L, r0, T = topo[b], lens[b], int(row_off[b]), Ts[b]
        x = inp[b]
        ref, rk, rv = orc.tree_attention(x.q, x.k_tree, x.v_tree, x.k_cache, x.v_cache, L, trees[t],
                                         SCALE, THETA)
        got = orc.bf16_to_f64(d_out[r0:r0 + T])
        assert np.abs(got - ref).max() <= ATOL_BF16, b
        np.testing.assert_array_equal(d_k[b][:, :L + T], rk[:, :L + T])
        np.testing.assert_array_equal(d_v[b][:, :L + T], rv[:, :L + T])
        done[r0:r0 + T] = True
    assert (d_out[~done] == fill_bits).all()
    for b in (1, 2, 3, 5):
        np.testing.assert_array_equal(d_k[b], inp[b].k_cache)
        np.testing.assert_array_equal(d_v[b], inp[b].v_cache)


def accept_inputs(trees, bank, topo, seed):
    g = np.random.default_rng(seed)
    rows = sum(bank.T[t] for t in topo)
    V = 50
    am = g.integers(0, V, rows).astype(np.int32)
    p1 = g.random(rows).astype(np.float32)
    toks, row = [], 0
    for b, t in enumerate(topo):
        T = bank.T[t]
        pa = [0.0, 1.0, 0.7, 0.9, 0.5, 0.3][b % 6]
        toks.append(synth.draft_tokens(trees[t], am[row:row + T], g.random(T), g.integers(0, V, T), pa))
        row += T
    return np.concatenate(toks).astype(np.int32), am, p1


def test_accept_device_arrays_equal_host_arrays(api, trees):
    bank = api.Bank(trees)
    topo = [4, 1, 0, 2, 3, 4, 1, 2]
    B = len(topo)
    tok, am, p1 = accept_inputs(trees, bank, topo, 29)
    cap_path = max(bank.D) + 2

    def outs():
        return (torch.full((B,), -7, dtype=torch.int32, device="cuda"),
                torch.full((B, cap_path), -7, dtype=torch.int32, device="cuda"),
                torch.full((B,), -7, dtype=torch.int32, device="cuda"),
                torch.zeros(B, device="cuda"))

    a1, path1, bon1, best1 = outs()
    api.accept_batched(bank, topo, dev_i32(tok), dev_i32(am), torch.from_numpy(p1).cuda(), a1, path1,
                       bon1, best1)
    a2, path2, bon2, best2 = outs()
    row_off = np.concatenate([[0], np.cumsum([bank.T[t] for t in topo])]).astype(np.int32)
    api.accept_batched_device(bank, dev_i32(np.asarray(topo, np.int32)), dev_i32(row_off), dev_i32(tok),
                              dev_i32(am), torch.from_numpy(p1).cuda(), a2, path2, bon2, best2)
    torch.cuda.synchronize()
    for x, y in ((a1, a2), (path1, path2), (bon1, bon2), (best1, best2)):
        np.testing.assert_array_equal(x.cpu().numpy(), y.cpu().numpy())
    # and the oracle, sequence by sequence
    a, path, bon = a2.cpu().numpy(), path2.cpu().numpy(), bon2.cpu().numpy()
    for b, t in enumerate(topo):
        r0, T = int(row_off[b]), bank.T[t]
        ra, rpath, rbonus, _ = orc.accept(trees[t], tok[r0:r0 + T], am[r0:r0 + T])
        assert (a[b], bon[b]) == (ra, rbonus)
        assert path[b, : ra + 1].tolist() == list(rpath)


def test_accept_device_arrays_invalid_entries(api, trees):
    """A tree index outside the bank, a row range shorter than the tree, a
    tree deeper than the path rows hold and rows past the capacity: accept
    length, bonus and path -1; the valid sequence is accepted as the oracle
    does."""
    bank = api.Bank(trees)
    T0, T1 = bank.T[2], bank.T[1]
    topo = np.array([2, len(trees), 1, 4, 0, 4], np.int32)
    rows_cap = T0 + T1 + 200
    # sequence 5's rows start 100 below 2^31 (their end does not fit in int32)
    row_off = np.array([0, T0, T0 + 1, T0 + T1, rows_cap - 4, 2**31 - 100, 2**31 - 1], np.int32)
    tok_v, am_v, p1_v = accept_inputs(trees, bank, [2], 31)
    tok = np.zeros(rows_cap, np.int32)
    am = np.zeros(rows_cap, np.int32)
    p1 = np.zeros(rows_cap, np.float32)
    tok[:T0], am[:T0], p1[:T0] = tok_v, am_v, p1_v
    B = len(topo)
    cap_path = bank.D[2] + 1          # tree 4 (sequence 3) is deeper: not verified
    assert bank.D[4] + 1 > cap_path and bank.D[0] + 1 <= cap_path
    assert row_off[4] - row_off[3] >= bank.T[4]
    a = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    path = torch.full((B, cap_path), -7, dtype=torch.int32, device="cuda")
    bon = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    best = torch.full((B,), 3.0, device="cuda")
    api.accept_batched_device(bank, dev_i32(topo), dev_i32(row_off), dev_i32(tok), dev_i32(am),
                              torch.from_numpy(p1).cuda(), a, path, bon, best)
    torch.cuda.synchronize()
    a, path, bon, best = a.cpu().numpy(), path.cpu().numpy(), bon.cpu().numpy(), best.cpu().numpy()
    ra, rpath, rbonus, rbest = orc.accept(trees[2], tok_v, am_v)
    assert (a[0], bon[0]) == (ra, rbonus)
    assert path[0, : ra + 1].tolist() == list(rpath)
    assert best[0] == p1_v[rbest]
    for b in range(1, B):
        assert a[b] == -1 and bon[b] == -1 and best[b] == 0.0, b
        assert (path[b] == -1).all(), b


def test_compact_device_arrays_equal_host_arrays(api, trees):
    g = np.random.default_rng(37)
    B, n_layers, Hkv, d = 5, 2, 4, 128
    lens = [0, 50, 7, 300, 129]
    topo = [4, 0, 2, 3, 1]
    cap = max(lens) + 128 + 4
    caches = [synth.f32_to_bf16_bits(g.standard_normal((2, n_layers, Hkv, cap, d)).astype(np.float32))
              for _ in range(B)]
    cap_path = 8
    paths = np.full((B, cap_path), -1, np.int32)
    acc = np.zeros(B, np.int32)
    for b, t in enumerate(topo):
        T = len(trees[t])
        am = g.integers(0, 3, T)
        tok = synth.draft_tokens(trees[t], am, g.random(T), g.integers(0, 3, T), 0.8)
        a, path, _, _ = orc.accept(trees[t], tok, am)
        acc[b] = a
        paths[b, : a + 1] = path
    k1 = [dev_bf16(c[0]) for c in caches]
    v1 = [dev_bf16(c[1]) for c in caches]
    api.kv_compact_batched(dev_i32(paths), dev_i32(acc), lens, k1, v1)
    lens_d = list(lens)
    lens_d[3] = -1                     # prefix lengths outside [0, cap): left alone
    lens_d[1] = 2**31 - 2
    k2 = [dev_bf16(c[0]) for c in caches]
    v2 = [dev_bf16(c[1]) for c in caches]
    api.kv_compact_batched_device(dev_i32(paths), dev_i32(acc), dev_i32(np.asarray(lens_d, np.int32)),
                                  k2, v2)
    torch.cuda.synchronize()
    for b in range(B):
        if b in (1, 3):
            np.testing.assert_array_equal(host_bits(k2[b]), caches[b][0])
            np.testing.assert_array_equal(host_bits(v2[b]), caches[b][1])
        else:
            np.testing.assert_array_equal(host_bits(k2[b]), host_bits(k1[b]))
            np.testing.assert_array_equal(host_bits(v2[b]), host_bits(v1[b]))
