"""GPU: the allocation-free attention entry point (entmtp_tree_attn_noalloc)
against entmtp_tree_attn with a caller workspace.

Both run the same kernels, so outputs and cache appends must agree bit for
bit; the first case is also held to the oracle's bar (attention within 2e-2
of the fp64 reference, bit-exact cache append).  Two no-alloc calls run back
to back before anything is compared, the second smaller than the first (the
shared static array keeps the first call's contents).  A call whose
workspace bound exceeds the static array is rejected on the host.
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import entmtp_oracle as orc  # noqa: E402
from paper_2606_27550_amd import synth  # noqa: E402
from tests.helpers import dev_bf16, host_bits  # noqa: E402

pytestmark = pytest.mark.gpu

ATOL_BF16 = 2e-2
THETA = 10000.0
D = 128


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


def say(*a):
    print("[gpu-test]", *a, flush=True)


def case(seed, T, depth, L, Hq, Hkv):
    parent = synth.uniform_attach_tree(seed, T, depth) if T > 1 else [-1]
    inp = synth.attn_inputs(seed, T, Hq, Hkv, D, L, L + T + 3)
    return parent, inp


def test_noalloc_matches_workspace_entry_point(api):
    # first the larger call (128 nodes, GQA 32:8, prefix 2048), then a
    # smaller one (27 nodes, 32 heads, prefix 256), both through the static
    # scratch, each into its own cache copy
    cases = [case(7, 128, 6, 2048, 32, 8), case(8, 27, 4, 256, 32, 32)]
    scale = 1 / math.sqrt(D)
    runs = []
    for parent, inp in cases:
        bank = api.Bank([parent])
        T, Hq, Hkv = len(parent), inp.q.shape[1], inp.k_tree.shape[1]
        L = inp.k_cache.shape[1] - T - 3
        need = api.tree_attn_workspace(T, Hq, Hkv, D, L)
        assert 0 < need <= api.NOALLOC_SCRATCH_BYTES, need
        runs.append({"bank": bank, "inp": inp, "parent": parent, "T": T, "L": L,
                     "q": dev_bf16(inp.q), "kt": dev_bf16(inp.k_tree), "vt": dev_bf16(inp.v_tree),
                     "kc": dev_bf16(inp.k_cache), "vc": dev_bf16(inp.v_cache),
                     "out": torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")})
    for r in runs:   # two no-alloc calls in a row, the second smaller
        say(f"noalloc call: T {r['T']} prefix {r['L']}")
        api.tree_attn_noalloc(r["bank"], 0, r["q"], r["kt"], r["vt"], r["kc"], r["vc"], r["L"], scale,
                              THETA, r["out"])
    torch.cuda.synchronize()
    for r in runs:   # the same calls with a caller workspace, into fresh caches
        inp = r["inp"]
        T, Hq, Hkv = r["T"], inp.q.shape[1], inp.k_tree.shape[1]
        kc2, vc2 = dev_bf16(inp.k_cache), dev_bf16(inp.v_cache)
        out2 = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(api.tree_attn_workspace(T, Hq, Hkv, D, r["L"]), dtype=torch.uint8,
                         device="cuda")
        api.tree_attn(r["bank"], 0, r["q"], r["kt"], r["vt"], kc2, vc2, r["L"], scale, THETA, out2, ws)
        torch.cuda.synchronize()
        assert torch.equal(r["out"].view(torch.int16), out2.view(torch.int16))
        assert torch.equal(r["kc"].view(torch.int16), kc2.view(torch.int16))
        assert torch.equal(r["vc"].view(torch.int16), vc2.view(torch.int16))
    # the oracle's bar on the smaller call
    r = runs[1]
    inp = r["inp"]
    ref, rk, rv = orc.tree_attention(inp.q, inp.k_tree, inp.v_tree, inp.k_cache, inp.v_cache, r["L"],
                                     r["parent"], scale, THETA)
    err = float(np.abs(r["out"].float().cpu().numpy() - ref).max())
    say(f"  27-node call vs oracle: max abs err {err:.2e}")
    assert err <= ATOL_BF16
    n = r["L"] + r["T"]
    np.testing.assert_array_equal(host_bits(r["kc"])[:, :n], rk[:, :n])
    np.testing.assert_array_equal(host_bits(r["vc"])[:, :n], rv[:, :n])


def test_noalloc_rejects_sizes_beyond_the_scratch(api):
    # a 256-node tree at prefix 8192 with 64 heads: its workspace bound
    # (132 MiB) is larger than the static array, so the call returns ENOSPC
    # on the host and launches nothing
    T, L, H = 256, 8192, 64
    parent = synth.uniform_attach_tree(9, T, 8)
    bank = api.Bank([parent])
    assert api.tree_attn_workspace(T, H, H, D, L) > api.NOALLOC_SCRATCH_BYTES
    cap = L + T
    kc = torch.zeros((H, cap, D), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    q = torch.zeros((T, H, D), dtype=torch.bfloat16, device="cuda")
    kt = torch.zeros((T, H, D), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros_like(q)
    with pytest.raises(api.EntmtpError) as e:
        api.tree_attn_noalloc(bank, 0, q, kt, kt, kc, vc, L, 0.1, THETA, out)
    assert e.value.code == api.ENOSPC
    assert "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert not out.any()   # nothing ran
