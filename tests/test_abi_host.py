"""Host-side checks of the C ABI (no GPU): the library loads and exports every
symbol the header declares, the bank planner's image equals the oracle's
buffers bit for bit, validation errors come back as the documented status
codes, and the ladder policy matches the oracle."""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

from oracle import entmtp_oracle as orc
from paper_2606_27550_amd import api, synth
from tests.conftest import ROOT, golden
from tests.test_oracle_bank import all_parent_arrays


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "entmtp.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(entmtp_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    syms = declared_symbols()
    assert len(syms) >= 14
    lib = ctypes.CDLL(api.LIB_PATH)
    for s in syms:
        assert hasattr(lib, s), s
    assert set(syms) == set(api._SIGNATURES), "binding and header disagree"


def check_entry(bank, k, parent):
    e = bank.export(k)
    ref = orc.bank_entry(parent)
    assert e["T"] == ref["T"] and e["D"] == ref["D"]
    np.testing.assert_array_equal(e["mask"], ref["mask"])
    np.testing.assert_array_equal(e["depth"], ref["depth"])
    np.testing.assert_array_equal(e["path"], ref["path"])
    np.testing.assert_array_equal(e["retrieve"], ref["retrieve"])
    np.testing.assert_array_equal(e["leaves"], ref["leaves"])
    np.testing.assert_array_equal(e["parent"], np.asarray(parent))


def test_bank_matches_oracle_on_all_small_trees():
    trees = [p for T in range(1, 7) for p in all_parent_arrays(T)]
    bank = api.Bank(trees, device=None)
    assert api.lib.entmtp_bank_size(bank.handle) == len(trees)
    for k, p in enumerate(trees):
        check_entry(bank, k, p)


def test_bank_matches_oracle_on_workload_trees():
    trees = []
    for wl in synth.WORKLOADS.values():
        trees += synth.workload_trees(wl)
    trees += [synth.chain_tree(32), synth.star_tree(256), [-1]]
    rng = np.random.default_rng(5)
    trees += [[-1] + [int(rng.integers(0, i)) for i in range(1, 200)]]
    bank = api.Bank(trees, device=None)
    for k, p in enumerate(trees):
        check_entry(bank, k, p)
    assert bank.T[:5] == [27, 1, 8, 26, 64]


@pytest.mark.parametrize("parents,code", [
    ([[-1, 0, 2]], api.ETREE), ([[0, 0]], api.ETREE), ([[-1, -1]], api.ETREE),
    ([[-1, 0], [-1, 1]], api.ETREE), ([[-1] + [0] * 256], api.ERANGE),
    ([[-1] + list(range(32))], api.ERANGE), ([[]], api.ERANGE), ([], api.EINVAL)])
def test_bank_errors(parents, code):
    with pytest.raises(api.EntmtpError) as ei:
        api.Bank(parents, device=None)
    assert ei.value.code == code
    assert api.last_error()


def test_bank_limits_accepted():
    api.Bank([[-1] + [0] * 255, [-1] + list(range(31))], device=None)


def test_device_array_batched_calls_reject_bad_arguments_without_launching():
    """The batched calls that read their per-sequence choices from device
    memory check everything the host can see before any launch."""
    lib = api.lib
    host_bank = api.Bank([[-1, 0], [-1, 0, 0, 1]], device=None)
    p = ctypes.c_void_p(16)                      # never dereferenced: validation fails first
    ptrs = (ctypes.c_void_p * 2)(16, 16)
    nulls = (ctypes.c_void_p * 2)(16, None)
    for B in (0, api.B_MAX + 1):
        assert lib.entmtp_tree_attn_batched_device(host_bank.handle, B, p, p, p, 8, p, p, p, ptrs, ptrs,
                                                   100, 32, 8, 128, 0.1, 0.0, p, p, 1 << 20,
                                                   None) == api.EINVAL
        assert lib.entmtp_accept_batched_device(host_bank.handle, B, p, p, 8, p, p, None, p, p, 4, p,
                                                None, None) == api.EINVAL
        assert lib.entmtp_kv_compact_batched_device(B, p, 4, p, p, ptrs, ptrs, 1, 0, 8, 100, 128,
                                                    None) == api.EINVAL
    rc = lib.entmtp_tree_attn_batched_device(host_bank.handle, 2, p, p, p, 8, p, p, p, ptrs, ptrs, 100,
                                             32, 8, 128, 0.1, 0.0, p, p, 1 << 20, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    rc = lib.entmtp_accept_batched_device(host_bank.handle, 2, p, p, 8, p, p, None, p, p, 4, p, None,
                                          None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    # compaction needs no bank: its device arrays and host cache lists
    assert lib.entmtp_kv_compact_batched_device(2, p, 4, p, None, ptrs, ptrs, 1, 0, 8, 100, 128,
                                                None) == api.EINVAL
    assert lib.entmtp_kv_compact_batched_device(2, p, 4, p, p, ptrs, nulls, 1, 0, 8, 100, 128,
                                                None) == api.EINVAL
    assert lib.entmtp_kv_compact_batched_device(2, p, 4, p, p, ptrs, ptrs, 1, 0, 8, 100, 12,
                                                None) == api.EINVAL
    assert lib.entmtp_kv_compact_batched_device(2, p, 0, p, p, ptrs, ptrs, 1, 0, 8, 100, 128,
                                                None) == api.EINVAL
    # the workspace bound: zero for invalid arguments, per sequence for a batch
    ws = api.tree_attn_batched_device_workspace
    assert ws(host_bank, 0, 32, 8, 128, 4096) == 0
    assert ws(host_bank, api.B_MAX + 1, 32, 8, 128, 4096) == 0
    assert ws(host_bank, 2, 30, 8, 128, 4096) == 0
    assert ws(host_bank, 2, 32, 8, 64, 4096) == 0
    assert ws(host_bank, 2, 32, 8, 128, 0) == 0
    one = ws(host_bank, 1, 32, 8, 128, 4096)
    assert one > 0
    assert one * 4 - 2 * 256 <= ws(host_bank, 4, 32, 8, 128, 4096) <= 4 * one
    assert ws(host_bank, 1, 32, 8, 128, 8192) >= one


def test_kernel_calls_reject_bad_arguments_without_launching():
    lib = api.lib
    host_bank = api.Bank([[-1, 0]], device=None)
    p = ctypes.c_void_p(16)                      # never dereferenced: validation fails first
    # host-only bank cannot drive kernels
    rc = lib.entmtp_accept(host_bank.handle, 0, p, p, None, p, p, p, None, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    rc = lib.entmtp_tree_attn(host_bank.handle, 0, p, p, p, p, p, 100, 0, 32, 32, 128, 0.1, 0.0,
                              p, p, 1 << 20, None)
    assert rc == api.EINVAL
    # sizes
    assert lib.entmtp_verify_logits(p, p, 0, 4096, 32000, p, None) == api.EINVAL
    assert lib.entmtp_verify_logits(p, p, 27, 4100 + 2, 32000, p, None) == api.EINVAL
    assert lib.entmtp_verify_logits(None, p, 27, 4096, 32000, p, None) == api.EINVAL
    assert lib.entmtp_logit_stats(p, 27, 32000, 0.0, p, p, p, None) == api.EINVAL
    assert lib.entmtp_logit_stats(p, 0, 32000, 1.0, p, p, p, None) == api.EINVAL
    assert lib.entmtp_kv_compact(p, 5, p, 10, p, p, 1, 0, 32, 100, 12, None) == api.EINVAL
    assert lib.entmtp_kv_compact(p, 0, p, 10, p, p, 1, 0, 32, 100, 128, None) == api.EINVAL
    assert lib.entmtp_kv_compact(p, 5, p, -1, p, p, 1, 0, 32, 100, 128, None) == api.EINVAL
    assert lib.entmtp_kv_compact(p, 5, p, 10, p, p, 2, 5, 32, 100, 128, None) == api.EINVAL
    # fused LM head + statistics and its two halves
    assert lib.entmtp_verify_logits_stats(p, p, 27, 4100, 32000, 1.0, p, p, p, p, p, 1 << 20,
                                          None) == api.EINVAL
    assert lib.entmtp_verify_logits_partials(p, p, 27, 264, 32000, 1.0, p, p, 1 << 20,
                                             None) == api.EINVAL
    assert lib.entmtp_verify_logits_partials(p, p, 27, 4096, 32000, 0.0, p, p, 1 << 20,
                                             None) == api.EINVAL
    assert lib.entmtp_verify_logits_partials(p, p, 27, 4096, 32000, 1.0, p, p, 16,
                                             None) == api.ENOSPC
    assert lib.entmtp_stats_finalize(None, 27, 32000, 1.0, p, p, p, None) == api.EINVAL
    assert lib.entmtp_stats_finalize(p, 27, 32000, float("inf"), p, p, p, None) == api.EINVAL
    assert api.stats_partials_bytes(27, 264, 32000) == 0
    assert api.stats_partials_bytes(27, 4096, 32000) >= 27 * 256 * 16
    assert api.verify_logits_stats_workspace(27, 264, 32000) > 0
    assert api.verify_logits_stats_workspace(27, 4096, 32000) == api.stats_partials_bytes(27, 4096, 32000)
    # batched calls: sizes and host arrays are checked before the bank
    two = (ctypes.c_int32 * 2)(0, 0)
    ptrs = (ctypes.c_void_p * 2)(16, 16)
    for B in (0, api.B_MAX + 1):
        assert lib.entmtp_tree_attn_batched(host_bank.handle, B, two, two, p, p, p, ptrs, ptrs, 100,
                                            32, 8, 128, 0.1, 0.0, p, p, 1 << 20, None) == api.EINVAL
        assert lib.entmtp_accept_batched(host_bank.handle, B, two, p, p, None, p, p, 4, p, None,
                                         None) == api.EINVAL
        assert lib.entmtp_kv_compact_batched(B, p, 4, p, two, ptrs, ptrs, 1, 0, 8, 100, 128,
                                             None) == api.EINVAL
    assert lib.entmtp_tree_attn_batched(host_bank.handle, 2, None, two, p, p, p, ptrs, ptrs, 100,
                                        32, 8, 128, 0.1, 0.0, p, p, 1 << 20, None) == api.EINVAL
    rc = lib.entmtp_tree_attn_batched(host_bank.handle, 2, two, two, p, p, p, ptrs, ptrs, 100, 32, 8,
                                      128, 0.1, 0.0, p, p, 1 << 20, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    assert lib.entmtp_accept_batched(host_bank.handle, 2, two, p, p, None, p, p, 0, p, None,
                                     None) == api.EINVAL
    neg = (ctypes.c_int32 * 2)(0, -1)
    assert lib.entmtp_kv_compact_batched(2, p, 4, p, neg, ptrs, ptrs, 1, 0, 8, 100, 128,
                                         None) == api.EINVAL
    nulls = (ctypes.c_void_p * 2)(16, None)
    assert lib.entmtp_kv_compact_batched(2, p, 4, p, two, ptrs, nulls, 1, 0, 8, 100, 128,
                                         None) == api.EINVAL
    assert api.tree_attn_batched_workspace(8, 128, 32, 8, 128, 16384) == \
        8 * api.tree_attn_workspace(128, 32, 8, 128, 16384)
    assert api.tree_attn_batched_workspace(0, 128, 32, 8, 128, 16384) == 0
    # typical acceptance: scalars and pointers before the bank
    f = ctypes.c_float
    assert lib.entmtp_draft_logits(host_bank.handle, 0, p, p, 260, 100, p, p, p, p, None) == api.EINVAL
    assert lib.entmtp_draft_logits(host_bank.handle, 0, p, None, 256, 100, p, p, p, p,
                                   None) == api.EINVAL
    assert lib.entmtp_draft_logits(host_bank.handle, 0, p, p, 256, 0, p, p, p, p, None) == api.EINVAL
    rc = lib.entmtp_draft_logits(host_bank.handle, 0, p, p, 256, 100, p, p, p, p, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    for it, eps, alpha in ((0.0, 0.09, 0.3), (float("inf"), 0.09, 0.3), (1.0, -0.1, 0.3),
                           (1.0, 0.09, float("nan")), (1.0, float("inf"), 0.3)):
        assert lib.entmtp_accept_typical(host_bank.handle, 0, p, p, p, p, p, p, f(it), f(eps), f(alpha),
                                         p, p, p, None, None) == api.EINVAL
    assert lib.entmtp_accept_typical(host_bank.handle, 0, p, p, p, p, None, p, f(1.0), f(0.09),
                                     f(0.3), p, p, p, None, None) == api.EINVAL
    rc = lib.entmtp_accept_typical(host_bank.handle, 0, p, p, p, p, p, p, f(1.0), f(0.09), f(0.3),
                                   p, p, p, None, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    # frontier scoring: sizes and inputs before the bank
    u8 = ctypes.c_void_p(16)
    assert lib.entmtp_frontier_score(host_bank.handle, 0, u8, 0, u8, None, None, p, p, None) == api.EINVAL
    assert lib.entmtp_frontier_score(host_bank.handle, 0, u8, 4, None, p, None, p, p, None) == api.EINVAL
    assert lib.entmtp_frontier_score(host_bank.handle, 0, None, 4, u8, None, None, p, p, None) == api.EINVAL
    rc = lib.entmtp_frontier_score(host_bank.handle, 0, u8, 4, u8, None, None, p, p, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    # stochastic acceptance
    fs = ctypes.c_float
    assert lib.entmtp_accept_stochastic(host_bank.handle, 0, p, p, p, 0, fs(1.0), p, p, p, p, p, p,
                                        p, p, None) == api.EINVAL
    assert lib.entmtp_accept_stochastic(host_bank.handle, 0, p, p, p, 100, fs(0.0), p, p, p, p, p,
                                        p, p, p, None) == api.EINVAL
    assert lib.entmtp_accept_stochastic(host_bank.handle, 0, p, p, p, 100, fs(1.0), None, p, p, p,
                                        p, p, p, p, None) == api.EINVAL
    rc = lib.entmtp_accept_stochastic(host_bank.handle, 0, p, p, p, 100, fs(1.0), p, p, p, p, p, p,
                                      p, p, None)
    assert rc == api.EINVAL and "arena" in api.last_error()
    # workspace query
    assert api.tree_attn_workspace(27, 32, 32, 64, 256) == 0
    assert api.tree_attn_workspace(27, 30, 8, 128, 256) == 0
    assert api.tree_attn_workspace(0, 32, 32, 128, 256) == 0


def test_workspace_is_monotone():
    prev_t = 0
    for T in (1, 8, 26, 27, 32, 33, 64, 128, 200, 256):
        prev_l = 0
        for L in (0, 31, 32, 256, 2048, 4096, 9216, 16384, 100000):
            w = api.tree_attn_workspace(T, 32, 8, 128, L)
            assert w >= prev_l
            prev_l = w
        assert prev_l >= prev_t
        prev_t = prev_l


def test_ladder_matches_oracle():
    g = golden("ladder_trace.json")
    rung = 0
    for s, want in zip(g["s"], g["rungs"]):
        rung = api.ladder_next(rung, g["n_rungs"], s, g["tau_on"], g["tau_off"])
        assert rung == want
    rng = np.random.default_rng(0)
    r1 = r2 = 2
    for s in rng.random(5000):
        s = float(np.float32(s))
        r1 = api.ladder_next(r1, 5, s, 0.8, 0.6)
        r2 = orc.ladder_next(r2, 5, s, float(np.float32(0.8)), float(np.float32(0.6)))
        assert r1 == r2
    with pytest.raises(api.EntmtpError):
        api.ladder_next(5, 5, 0.5, 0.8, 0.6)
    with pytest.raises(api.EntmtpError):
        api.ladder_next(0, 5, 0.5, 0.6, 0.8)


def test_ladder_batched_matches_oracle():
    """One ladder per sequence, moved by one call: the hand-traced fixture in
    every lane, then 16 independent sequences over 2000 steps against the
    oracle, with s drawn on and next to both thresholds."""
    g = golden("ladder_trace.json")
    rung = np.zeros(4, np.int32)
    for s, want in zip(g["s"], g["rungs"]):
        api.ladder_next_batched(rung, np.full(4, s, np.float32), g["n_rungs"], g["tau_on"],
                                g["tau_off"])
        assert rung.tolist() == [want] * 4
    rng = np.random.default_rng(3)
    on, off = float(np.float32(0.8)), float(np.float32(0.6))
    edges = np.array([0.8, 0.6, np.nextafter(np.float32(0.8), np.float32(1)),
                      np.nextafter(np.float32(0.6), np.float32(0))], np.float32)
    rung = rng.integers(0, 5, 16).astype(np.int32)
    want = [int(r) for r in rung]
    for _ in range(2000):
        s = rng.random(16).astype(np.float32)
        pick = rng.random(16) < 0.2
        s[pick] = edges[rng.integers(0, 4, int(pick.sum()))]
        api.ladder_next_batched(rung, s, 5, 0.8, 0.6)
        want = [orc.ladder_next(w, 5, float(x), on, off) for w, x in zip(want, s)]
        assert rung.tolist() == want
    # an invalid rung anywhere leaves every rung unchanged
    bad = np.array([1, 2, 5, 0], np.int32)
    with pytest.raises(api.EntmtpError):
        api.ladder_next_batched(bad, np.ones(4, np.float32), 5, 0.8, 0.6)
    assert bad.tolist() == [1, 2, 5, 0]
    with pytest.raises(api.EntmtpError):
        api.ladder_next_batched(np.zeros(2, np.int32), np.ones(2, np.float32), 5, 0.6, 0.8)
    api.ladder_next_batched(np.zeros(0, np.int32), np.zeros(0, np.float32), 5, 0.8, 0.6)


def test_frontier_tree_matches_oracle():
    """entmtp_frontier_tree (the joint tree T u F, through the C ABI) against
    the oracle's NextChildren."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        n = int(rng.integers(1, 30))
        parent = [-1] + [int(rng.integers(0, i)) for i in range(1, n)]
        D = int(rng.integers(0, 8))
        joint, in_tree = api.frontier_tree(parent, D)
        ref, ref_in = orc.joint_tree(parent, D)
        assert joint == ref and in_tree == [int(x) for x in ref_in]


def test_frontier_tree_errors():
    import ctypes
    lib = api.lib
    parent = (ctypes.c_int32 * 4)(-1, 0, 0, 1)
    out = (ctypes.c_int32 * 8)()
    flags = (ctypes.c_uint8 * 8)()
    n = ctypes.c_int32(0)
    # depth 2 admits candidates under nodes 0, 1, 2 (depths 0, 1, 1): 7 nodes
    assert lib.entmtp_frontier_tree(parent, 4, 2, out, flags, 8, ctypes.byref(n)) == 0
    assert n.value == 7 and list(out[:7]) == [-1, 0, 0, 1, 0, 1, 2]
    assert list(flags[:7]) == [1, 1, 1, 1, 0, 0, 0]
    assert lib.entmtp_frontier_tree(parent, 4, 2, out, None, 6, ctypes.byref(n)) == api.ENOSPC
    assert n.value == 7
    bad = (ctypes.c_int32 * 3)(-1, 0, 2)       # a parent that does not precede its child
    assert lib.entmtp_frontier_tree(bad, 3, 2, out, flags, 8, ctypes.byref(n)) == api.EINVAL
    assert lib.entmtp_frontier_tree(parent, 4, -1, out, flags, 8, ctypes.byref(n)) == api.EINVAL
    assert lib.entmtp_frontier_tree(None, 4, 2, out, flags, 8, ctypes.byref(n)) == api.EINVAL


def test_step_config_layout_matches_header(tmp_path):
    """The binding's entmtp_step_config mirror has the header's field offsets
    and size (checked by compiling the header with the host C compiler)."""
    import ctypes
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    from paper_2606_27550_amd.api import StepConfig
    names = [f for f, _ in StepConfig._fields_]
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "entmtp.h"\nint main(void) {\n'
                   + "".join(f'  printf("%zu\\n", offsetof(entmtp_step_config, {n}));\n' for n in names)
                   + '  printf("%zu\\n", sizeof(entmtp_step_config));\n  return 0;\n}\n')
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [getattr(StepConfig, n).offset for n in names] + [ctypes.sizeof(StepConfig)]
    assert got == want
