"""ctypes binding of ``libentmtp.so``: argument marshalling only.

Every function here forwards to the C ABI declared in ``include/entmtp.h``
with the same name (minus the ``entmtp_`` prefix); all computation happens in
the library's HIP kernels.  Tensors are torch tensors on the GPU (bf16 ones as
``torch.bfloat16``); the stream defaults to torch's current stream.  Importing
this module fails if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libentmtp.so")

OK, EINVAL, ETREE, ERANGE, ENOSPC, EHIP, ETIMEDOUT = 0, -1, -2, -3, -4, -5, -6
T_MAX, D_MAX, MASK_WORDS, HEAD_DIM, B_MAX = 256, 31, 8, 128, 16

_c_i32, _c_i64, _c_f32, _c_sz, _c_p = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                       ctypes.c_size_t, ctypes.c_void_p)

class StepConfig(ctypes.Structure):
    """entmtp_step_config, field for field."""
    _fields_ = [("n_layers", _c_i32), ("Hq", _c_i32), ("Hkv", _c_i32), ("d", _c_i32),
                ("cap", _c_i32), ("tree_rows", _c_i32), ("scale", _c_f32), ("rope_theta", _c_f32),
                ("k_cache", _c_p), ("v_cache", _c_p), ("cache_layer_stride", _c_i64),
                ("w_lm", _c_p), ("hid", _c_i32), ("V", _c_i32), ("inv_temp", _c_f32),
                ("logits", _c_p), ("entropy", _c_p), ("top1p", _c_p), ("argmax", _c_p),
                ("accept_len", _c_p), ("bonus", _c_p), ("best_top1p", _c_p), ("path", _c_p),
                ("path_capacity", _c_i32), ("workspace", _c_p), ("workspace_bytes", _c_sz),
                ("stream", _c_p), ("tau_on", _c_f32), ("tau_off", _c_f32),
                ("device_prefix_fixed", _c_i32)]


# name -> (restype, argtypes), mirroring include/entmtp.h
_SIGNATURES = {
    "entmtp_last_error": (ctypes.c_char_p, []),
    "entmtp_version": (ctypes.c_char_p, []),
    "entmtp_bank_build": (_c_i32, [_c_p, _c_p, _c_i32, _c_p, _c_sz, ctypes.POINTER(_c_sz), _c_p,
                                   ctypes.POINTER(_c_p)]),
    "entmtp_bank_destroy": (_c_i32, [_c_p]),
    "entmtp_bank_size": (_c_i32, [_c_p]),
    "entmtp_bank_info": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p]),
    "entmtp_bank_export": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "entmtp_tree_attn_workspace": (_c_sz, [_c_i32, _c_i32, _c_i32, _c_i32, _c_i32]),
    "entmtp_tree_attn": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32, _c_i32,
                                  _c_i32, _c_i32, _c_i32, _c_f32, _c_f32, _c_p, _c_p, _c_sz, _c_p]),
    "entmtp_tree_attn_noalloc": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32,
                                          _c_i32, _c_i32, _c_i32, _c_i32, _c_f32, _c_f32, _c_p,
                                          _c_p]),
    "entmtp_tree_attn_batched_workspace": (_c_sz, [_c_i32] * 6),
    "entmtp_tree_attn_batched": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p,
                                          _c_i32, _c_i32, _c_i32, _c_i32, _c_f32, _c_f32, _c_p, _c_p,
                                          _c_sz, _c_p]),
    "entmtp_tree_attn_batched_device_workspace": (_c_sz, [_c_p] + [_c_i32] * 5),
    "entmtp_tree_attn_batched_device": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_i32, _c_p, _c_p,
                                                 _c_p, _c_p, _c_p, _c_i32, _c_i32, _c_i32, _c_i32,
                                                 _c_f32, _c_f32, _c_p, _c_p, _c_sz, _c_p]),
    "entmtp_accept_batched": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i32,
                                       _c_p, _c_p, _c_p]),
    "entmtp_accept_batched_device": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_i32, _c_p, _c_p, _c_p,
                                              _c_p, _c_p, _c_i32, _c_p, _c_p, _c_p]),
    "entmtp_kv_compact_batched": (_c_i32, [_c_i32, _c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_i32,
                                           _c_i64, _c_i32, _c_i32, _c_i32, _c_p]),
    "entmtp_kv_compact_batched_device": (_c_i32, [_c_i32, _c_p, _c_i32, _c_p, _c_p, _c_p, _c_p,
                                                  _c_i32, _c_i64, _c_i32, _c_i32, _c_i32, _c_p]),
    "entmtp_verify_logits": (_c_i32, [_c_p, _c_p, _c_i32, _c_i32, _c_i32, _c_p, _c_p]),
    "entmtp_logit_stats": (_c_i32, [_c_p, _c_i32, _c_i32, _c_f32, _c_p, _c_p, _c_p, _c_p]),
    "entmtp_verify_logits_stats_workspace": (_c_sz, [_c_i32, _c_i32, _c_i32]),
    "entmtp_stats_partials_bytes": (_c_sz, [_c_i32, _c_i32, _c_i32]),
    "entmtp_verify_logits_partials": (_c_i32, [_c_p, _c_p, _c_i32, _c_i32, _c_i32, _c_f32, _c_p, _c_p,
                                               _c_sz, _c_p]),
    "entmtp_stats_finalize": (_c_i32, [_c_p, _c_i32, _c_i32, _c_f32, _c_p, _c_p, _c_p, _c_p]),
    "entmtp_verify_logits_stats": (_c_i32, [_c_p, _c_p, _c_i32, _c_i32, _c_i32, _c_f32, _c_p, _c_p, _c_p,
                                            _c_p, _c_p, _c_sz, _c_p]),
    "entmtp_accept": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "entmtp_draft_logits": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_i32, _c_i32, _c_p, _c_p, _c_p, _c_p,
                                     _c_p]),
    "entmtp_accept_typical": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_f32,
                                       _c_f32, _c_f32, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "entmtp_frontier_tree": (_c_i32, [_c_p, _c_i32, _c_i32, _c_p, _c_p, _c_i32, ctypes.POINTER(_c_i32)]),
    "entmtp_frontier_score": (_c_i32, [_c_p, _c_i32, _c_p, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p,
                                       _c_p]),
    "entmtp_accept_stochastic": (_c_i32, [_c_p, _c_i32, _c_p, _c_p, _c_p, _c_i32, _c_f32, _c_p,
                                          _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "entmtp_kv_compact": (_c_i32, [_c_p, _c_i32, _c_p, _c_i32, _c_p, _c_p, _c_i32, _c_i64, _c_i32,
                                   _c_i32, _c_i32, _c_p]),
    "entmtp_ladder_next": (_c_i32, [_c_i32, _c_i32, _c_f32, _c_f32, _c_f32]),
    "entmtp_ladder_next_batched": (_c_i32, [_c_i32, _c_p, _c_p, _c_i32, _c_f32, _c_f32]),
    "entmtp_step_workspace": (_c_sz, [_c_p, ctypes.POINTER(StepConfig)]),
    "entmtp_step_create": (_c_i32, [_c_p, ctypes.POINTER(StepConfig), ctypes.POINTER(_c_p)]),
    "entmtp_step_destroy": (None, [_c_p]),
    "entmtp_step_launch": (_c_i32, [_c_p, _c_i32, _c_i32, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p,
                                    _c_p, _c_p]),
    "entmtp_step_arm": (_c_i32, [_c_p, _c_p, _c_p, _c_i32, _c_p, _c_p]),
    "entmtp_step_flush": (_c_i32, [_c_p]),
    "entmtp_step_wait": (_c_i32, [_c_p, ctypes.POINTER(_c_i32), ctypes.POINTER(_c_i32),
                                  ctypes.POINTER(_c_f32), ctypes.c_double]),
    "entmtp_step_device_start": (_c_i32, [_c_p, _c_i32, _c_i32]),
    "entmtp_step_launch_device": (_c_i32, [_c_p] * 9 + [_c_i32, _c_p, _c_p]),
    "entmtp_step_device_graph": (_c_i32, [_c_p, _c_i32] + [_c_p] * 8 + [_c_i32, _c_p]),
    "entmtp_step_graph_launch": (_c_i32, [_c_p, _c_p]),
    "entmtp_step_graph_destroy": (None, [_c_p]),
}


def _hip_runtimes():
    try:
        with open("/proc/self/maps") as f:
            return sorted({l.split()[-1] for l in f if "libamdhip64" in l})
    except OSError:
        return []


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_2606_27550_amd.build`")
    # torch owns the device memory and streams handed to the library, so the
    # library must resolve to the HIP runtime torch already loaded (the
    # dynamic loader reuses it by soname when torch comes first).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(_LIB_PATH)
    rts = _hip_runtimes()
    if len(rts) > 1:
        raise ImportError("two HIP runtimes are loaded in this process "
                          f"({rts}); import torch before anything that loads libamdhip64")
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()
LIB_PATH = _LIB_PATH


class EntmtpError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"entmtp status {code}: {message}")
        self.code = code


def _check(rc: int) -> int:
    if rc < 0:
        raise EntmtpError(rc, lib.entmtp_last_error().decode())
    return rc


def last_error() -> str:
    return lib.entmtp_last_error().decode()


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _np_p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


# --------------------------------------------------------------------- bank --

class Bank:
    """TopologyBank: the trees' masks, depths, paths and retrieve rows in one
    device arena.  ``device=None`` builds a host-only bank (info / export
    only, no GPU involved)."""

    def __init__(self, trees: Sequence[Sequence[int]], device="cuda", stream=None):
        self.trees = [list(map(int, t)) for t in trees]
        parents = np.ascontiguousarray(np.concatenate([np.asarray(t, np.int32) for t in self.trees])
                                       if self.trees else np.zeros(0, np.int32))
        sizes = np.ascontiguousarray([len(t) for t in self.trees], dtype=np.int32)
        need = _c_sz(0)
        handle = _c_p(None)
        self._handle = None
        self.arena = None
        if device is None:
            _check(lib.entmtp_bank_build(_np_p(parents), _np_p(sizes), len(self.trees), None, 0,
                                         ctypes.byref(need), None, ctypes.byref(handle)))
        else:
            import torch
            _check(lib.entmtp_bank_build(_np_p(parents), _np_p(sizes), len(self.trees), None, 0,
                                         ctypes.byref(need), None, None))
            self.arena = torch.empty(max(int(need.value), 256), dtype=torch.uint8, device=device)
            _check(lib.entmtp_bank_build(_np_p(parents), _np_p(sizes), len(self.trees),
                                         _p(self.arena), self.arena.numel(), ctypes.byref(need),
                                         _stream(stream), ctypes.byref(handle)))
        self._handle = handle
        self.arena_bytes = int(need.value)
        self.T, self.D, self.n_leaves = [], [], []
        for k in range(len(self.trees)):
            T, D, nl = _c_i32(), _c_i32(), _c_i32()
            _check(lib.entmtp_bank_info(self._handle, k, ctypes.byref(T), ctypes.byref(D),
                                        ctypes.byref(nl)))
            self.T.append(T.value)
            self.D.append(D.value)
            self.n_leaves.append(nl.value)

    @property
    def handle(self):
        return self._handle

    def __len__(self):
        return len(self.trees)

    def export(self, topo: int) -> dict:
        T, D, nl = self.T[topo], self.D[topo], self.n_leaves[topo]
        mask = np.zeros((T, MASK_WORDS), np.uint32)
        depth = np.zeros(T, np.int32)
        path = np.zeros((T, D + 1), np.int32)
        retrieve = np.zeros((nl, D + 1), np.int32)
        parent = np.zeros(T, np.int32)
        _check(lib.entmtp_bank_export(self._handle, topo, _np_p(mask), _np_p(depth), _np_p(path),
                                      _np_p(retrieve), _np_p(parent)))
        return {"T": T, "D": D, "mask": mask, "depth": depth, "path": path,
                "retrieve": retrieve, "parent": parent,
                "leaves": np.array([row[row >= 0][-1] for row in retrieve], np.int32)}

    def close(self):
        if self._handle is not None and self._handle.value:
            lib.entmtp_bank_destroy(self._handle)
        self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------------------ kernels --

def _need(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


def _dev(t, name, dtype, shape=None, min_numel=None):
    """Host-side check that a tensor is what the kernel will assume."""
    import torch
    _need(isinstance(t, torch.Tensor), f"{name} must be a torch tensor")
    _need(t.is_cuda, f"{name} must live on the GPU")
    _need(t.dtype == dtype, f"{name} must be {dtype}, got {t.dtype}")
    _need(t.is_contiguous(), f"{name} must be contiguous")
    if shape is not None:
        _need(tuple(t.shape) == tuple(shape), f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if min_numel is not None:
        _need(t.numel() >= min_numel, f"{name} needs at least {min_numel} elements")


def tree_attn_workspace(T: int, Hq: int, Hkv: int, d: int, prefix_len: int) -> int:
    return int(lib.entmtp_tree_attn_workspace(T, Hq, Hkv, d, prefix_len))


def tree_attn(bank: Bank, topo: int, q, k_tree, v_tree, k_cache, v_cache, prefix_len: int,
              scale: float, rope_theta: float, out, workspace, stream=None) -> None:
    """q [T,Hq,d], k_tree/v_tree [T,Hkv,d], caches [Hkv,cap,d], out [T,Hq,d] (bf16)."""
    import torch
    _need(0 <= topo < len(bank), "topo out of range")
    T = bank.T[topo]
    _need(q.dim() == 3 and k_cache.dim() == 3, "q and caches are 3-D")
    _, Hq, d = q.shape
    Hkv, cap, _ = k_cache.shape
    bf = torch.bfloat16
    _dev(q, "q", bf, (T, Hq, d))
    _dev(k_tree, "k_tree", bf, (T, Hkv, d))
    _dev(v_tree, "v_tree", bf, (T, Hkv, d))
    _dev(k_cache, "k_cache", bf, (Hkv, cap, d))
    _dev(v_cache, "v_cache", bf, (Hkv, cap, d))
    _dev(out, "out", bf, (T, Hq, d))
    _need(workspace.is_cuda and workspace.is_contiguous(), "workspace must be a contiguous GPU tensor")
    _check(lib.entmtp_tree_attn(bank.handle, topo, _p(q), _p(k_tree), _p(v_tree), _p(k_cache),
                                _p(v_cache), cap, prefix_len, Hq, Hkv, d, scale, rope_theta,
                                _p(out), _p(workspace), workspace.numel() * workspace.element_size(),
                                _stream(stream)))


NOALLOC_SCRATCH_BYTES = 96 * 1024 * 1024   # ENTMTP_NOALLOC_SCRATCH_BYTES


def tree_attn_noalloc(bank: Bank, topo: int, q, k_tree, v_tree, k_cache, v_cache, prefix_len: int,
                      scale: float, rope_theta: float, out, stream=None) -> None:
    """tree_attn without a workspace argument (the library's static scratch):
    for callers that cannot allocate; calls that can overlap on one device
    must be ordered by the caller."""
    import torch
    _need(0 <= topo < len(bank), "topo out of range")
    T = bank.T[topo]
    _need(q.dim() == 3 and k_cache.dim() == 3, "q and caches are 3-D")
    _, Hq, d = q.shape
    Hkv, cap, _ = k_cache.shape
    bf = torch.bfloat16
    _dev(q, "q", bf, (T, Hq, d))
    _dev(k_tree, "k_tree", bf, (T, Hkv, d))
    _dev(v_tree, "v_tree", bf, (T, Hkv, d))
    _dev(k_cache, "k_cache", bf, (Hkv, cap, d))
    _dev(v_cache, "v_cache", bf, (Hkv, cap, d))
    _dev(out, "out", bf, (T, Hq, d))
    _check(lib.entmtp_tree_attn_noalloc(bank.handle, topo, _p(q), _p(k_tree), _p(v_tree),
                                        _p(k_cache), _p(v_cache), cap, prefix_len, Hq, Hkv, d,
                                        scale, rope_theta, _p(out), _stream(stream)))


def _host_i32(values):
    a = np.ascontiguousarray(np.asarray(values, dtype=np.int32))
    return a, _np_p(a)


def _host_ptrs(tensors):
    arr = (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])
    return arr


def tree_attn_batched_workspace(B: int, T_max: int, Hq: int, Hkv: int, d: int,
                                max_prefix_len: int) -> int:
    return int(lib.entmtp_tree_attn_batched_workspace(B, T_max, Hq, Hkv, d, max_prefix_len))


def tree_attn_batched(bank: Bank, topo, prefix_len, q, k_tree, v_tree, k_caches, v_caches,
                      scale: float, rope_theta: float, out, workspace, stream=None) -> None:
    """Sequences' tree rows back to back in q [rows,Hq,d], k_tree/v_tree
    [rows,Hkv,d], out [rows,Hq,d]; one [Hkv,cap,d] cache pair per sequence."""
    import torch
    B = len(topo)
    _need(1 <= B <= B_MAX and len(prefix_len) == B and len(k_caches) == B and len(v_caches) == B,
          "topo, prefix_len and the cache lists need one entry per sequence")
    rows = sum(bank.T[t] for t in topo)
    Hq, d = q.shape[1], q.shape[2]
    Hkv = k_tree.shape[1]
    _dev(q, "q", torch.bfloat16, (rows, Hq, d))
    _dev(k_tree, "k_tree", torch.bfloat16, (rows, Hkv, d))
    _dev(v_tree, "v_tree", torch.bfloat16, (rows, Hkv, d))
    _dev(out, "out", torch.bfloat16, (rows, Hq, d))
    cap = k_caches[0].shape[1]
    for kc, vc in zip(k_caches, v_caches):
        _dev(kc, "k_cache", torch.bfloat16, (Hkv, cap, d))
        _dev(vc, "v_cache", torch.bfloat16, (Hkv, cap, d))
    _need(workspace.is_cuda and workspace.is_contiguous(), "workspace must be a contiguous GPU tensor")
    t_arr, t_p = _host_i32(topo)
    l_arr, l_p = _host_i32(prefix_len)
    kp, vp = _host_ptrs(k_caches), _host_ptrs(v_caches)
    _check(lib.entmtp_tree_attn_batched(bank.handle, B, t_p, l_p, _p(q), _p(k_tree), _p(v_tree), kp,
                                        vp, cap, Hq, Hkv, d, scale, rope_theta, _p(out),
                                        _p(workspace), workspace.numel() * workspace.element_size(),
                                        _stream(stream)))


def tree_attn_batched_device_workspace(bank: Bank, B: int, Hq: int, Hkv: int, d: int,
                                       cap: int) -> int:
    return int(lib.entmtp_tree_attn_batched_device_workspace(bank.handle, B, Hq, Hkv, d, cap))


def tree_attn_batched_device(bank: Bank, topo, prefix_len, row_off, q, k_tree, v_tree, k_caches,
                             v_caches, scale: float, rope_theta: float, out, workspace,
                             stream=None) -> None:
    """topo [B], prefix_len [B] and row_off [B+1]: int32 GPU tensors read by
    the kernels; q / k_tree / v_tree / out hold rows_cap = q.shape[0] rows;
    one [Hkv,cap,d] cache pair per sequence."""
    import torch
    B = len(k_caches)
    _need(1 <= B <= B_MAX and len(v_caches) == B, "one cache pair per sequence")
    _dev(topo, "topo", torch.int32, min_numel=B)
    _dev(prefix_len, "prefix_len", torch.int32, min_numel=B)
    _dev(row_off, "row_off", torch.int32, min_numel=B + 1)
    rows, Hq, d = q.shape
    Hkv = k_tree.shape[1]
    _dev(q, "q", torch.bfloat16, (rows, Hq, d))
    _dev(k_tree, "k_tree", torch.bfloat16, (rows, Hkv, d))
    _dev(v_tree, "v_tree", torch.bfloat16, (rows, Hkv, d))
    _dev(out, "out", torch.bfloat16, (rows, Hq, d))
    cap = k_caches[0].shape[1]
    for kc, vc in zip(k_caches, v_caches):
        _dev(kc, "k_cache", torch.bfloat16, (Hkv, cap, d))
        _dev(vc, "v_cache", torch.bfloat16, (Hkv, cap, d))
    _need(workspace.is_cuda and workspace.is_contiguous(), "workspace must be a contiguous GPU tensor")
    kp, vp = _host_ptrs(k_caches), _host_ptrs(v_caches)
    _check(lib.entmtp_tree_attn_batched_device(bank.handle, B, _p(topo), _p(prefix_len), _p(row_off),
                                               rows, _p(q), _p(k_tree), _p(v_tree), kp, vp, cap, Hq,
                                               Hkv, d, scale, rope_theta, _p(out), _p(workspace),
                                               workspace.numel() * workspace.element_size(),
                                               _stream(stream)))


def accept_batched_device(bank: Bank, topo, row_off, draft_tokens, argmax, top1p, accept_len, path,
                          bonus, best_top1p=None, stream=None) -> None:
    """topo [B] and row_off [B+1]: int32 GPU tensors; the per-node arrays hold
    rows_cap = draft_tokens.numel() rows; path is [B, path_capacity]."""
    import torch
    B = path.shape[0] if path.dim() == 2 else 0
    _need(1 <= B <= B_MAX, "path is [B, path_capacity] with 1 <= B <= 16")
    _dev(topo, "topo", torch.int32, min_numel=B)
    _dev(row_off, "row_off", torch.int32, min_numel=B + 1)
    _dev(draft_tokens, "draft_tokens", torch.int32)
    rows = draft_tokens.numel()
    _dev(argmax, "argmax", torch.int32, min_numel=rows)
    if top1p is not None:
        _dev(top1p, "top1p", torch.float32, min_numel=rows)
    _dev(accept_len, "accept_len", torch.int32, min_numel=B)
    _dev(bonus, "bonus", torch.int32, min_numel=B)
    if best_top1p is not None:
        _dev(best_top1p, "best_top1p", torch.float32, min_numel=B)
    _dev(path, "path", torch.int32)
    _check(lib.entmtp_accept_batched_device(bank.handle, B, _p(topo), _p(row_off), rows,
                                            _p(draft_tokens), _p(argmax), _p(top1p), _p(accept_len),
                                            _p(path), path.shape[1], _p(bonus), _p(best_top1p),
                                            _stream(stream)))


def kv_compact_batched_device(path, accept_len, prefix_len, k_caches, v_caches,
                              stream=None) -> None:
    """As kv_compact_batched with prefix_len [B] an int32 GPU tensor."""
    import torch
    B = len(k_caches)
    _need(1 <= B <= B_MAX and len(v_caches) == B, "one cache pair per sequence")
    _need(path.dim() == 2 and path.shape[0] == B, "path is [B, path_capacity]")
    _dev(path, "path", torch.int32)
    _dev(accept_len, "accept_len", torch.int32, min_numel=B)
    _dev(prefix_len, "prefix_len", torch.int32, min_numel=B)
    shape = k_caches[0].shape
    for kc, vc in zip(k_caches, v_caches):
        _need(kc.shape == shape and vc.shape == shape, "caches of equal shapes")
        _dev(kc, "k_cache", torch.bfloat16)
        _dev(vc, "v_cache", torch.bfloat16)
    if len(shape) == 3:
        n_layers, (Hkv, cap, d) = 1, shape
    else:
        n_layers, Hkv, cap, d = shape
    kp, vp = _host_ptrs(k_caches), _host_ptrs(v_caches)
    _check(lib.entmtp_kv_compact_batched_device(B, _p(path), path.shape[1], _p(accept_len),
                                                _p(prefix_len), kp, vp, n_layers, Hkv * cap * d,
                                                Hkv, cap, d, _stream(stream)))


def accept_batched(bank: Bank, topo, draft_tokens, argmax, top1p, accept_len, path, bonus,
                   best_top1p=None, stream=None) -> None:
    """Per-node arrays concatenated over sequences; path is [B, path_capacity]."""
    import torch
    B = len(topo)
    rows = sum(bank.T[t] for t in topo)
    _need(1 <= B <= B_MAX, "1 <= B <= 16")
    _dev(draft_tokens, "draft_tokens", torch.int32, min_numel=rows)
    _dev(argmax, "argmax", torch.int32, min_numel=rows)
    if top1p is not None:
        _dev(top1p, "top1p", torch.float32, min_numel=rows)
    _dev(accept_len, "accept_len", torch.int32, min_numel=B)
    _dev(bonus, "bonus", torch.int32, min_numel=B)
    if best_top1p is not None:
        _dev(best_top1p, "best_top1p", torch.float32, min_numel=B)
    _need(path.dim() == 2 and path.shape[0] == B, "path is [B, path_capacity]")
    _dev(path, "path", torch.int32)
    t_arr, t_p = _host_i32(topo)
    _check(lib.entmtp_accept_batched(bank.handle, B, t_p, _p(draft_tokens), _p(argmax), _p(top1p),
                                     _p(accept_len), _p(path), path.shape[1], _p(bonus),
                                     _p(best_top1p), _stream(stream)))


def kv_compact_batched(path, accept_len, prefix_len, k_caches, v_caches, stream=None) -> None:
    """path [B, path_capacity], accept_len [B] on the device; one cache pair per
    sequence, each [Hkv,cap,d] or [n_layers,Hkv,cap,d]."""
    import torch
    B = len(prefix_len)
    _need(1 <= B <= B_MAX and len(k_caches) == B and len(v_caches) == B,
          "one prefix length and cache pair per sequence")
    _need(path.dim() == 2 and path.shape[0] == B, "path is [B, path_capacity]")
    _dev(path, "path", torch.int32)
    _dev(accept_len, "accept_len", torch.int32, min_numel=B)
    shape = k_caches[0].shape
    for kc, vc in zip(k_caches, v_caches):
        _need(kc.shape == shape and vc.shape == shape, "caches of equal shapes")
        _dev(kc, "k_cache", torch.bfloat16)
        _dev(vc, "v_cache", torch.bfloat16)
    if len(shape) == 3:
        n_layers, (Hkv, cap, d) = 1, shape
    else:
        n_layers, Hkv, cap, d = shape
    l_arr, l_p = _host_i32(prefix_len)
    kp, vp = _host_ptrs(k_caches), _host_ptrs(v_caches)
    _check(lib.entmtp_kv_compact_batched(B, _p(path), path.shape[1], _p(accept_len), l_p, kp, vp,
                                         n_layers, Hkv * cap * d, Hkv, cap, d, _stream(stream)))


def verify_logits(hidden, w_lm, logits, stream=None) -> None:
    """hidden [T,hid] bf16, w_lm [V,hid] bf16 -> logits [T,V] fp32."""
    import torch
    _need(hidden.dim() == 2 and w_lm.dim() == 2, "hidden and w_lm are 2-D")
    T, hid = hidden.shape
    V = w_lm.shape[0]
    _dev(hidden, "hidden", torch.bfloat16, (T, hid))
    _dev(w_lm, "w_lm", torch.bfloat16, (V, hid))
    _dev(logits, "logits", torch.float32, (T, V))
    _check(lib.entmtp_verify_logits(_p(hidden), _p(w_lm), T, hid, V, _p(logits), _stream(stream)))


def verify_logits_stats_workspace(T: int, hid: int, V: int) -> int:
    return int(lib.entmtp_verify_logits_stats_workspace(T, hid, V))


def verify_logits_stats(hidden, w_lm, logits, inv_temp: float, entropy, top1p, argmax, workspace,
                        stream=None) -> None:
    """Fused LM head + statistics; same outputs as verify_logits then logit_stats."""
    import torch
    _need(hidden.dim() == 2 and w_lm.dim() == 2, "hidden and w_lm are 2-D")
    T, hid = hidden.shape
    V = w_lm.shape[0]
    _dev(hidden, "hidden", torch.bfloat16, (T, hid))
    _dev(w_lm, "w_lm", torch.bfloat16, (V, hid))
    _dev(logits, "logits", torch.float32, (T, V))
    for name, t, dt in (("entropy", entropy, torch.float32), ("top1p", top1p, torch.float32),
                        ("argmax", argmax, torch.int32)):
        if t is not None:
            _dev(t, name, dt, min_numel=T)
    _need(workspace.is_cuda and workspace.is_contiguous(), "workspace must be a contiguous GPU tensor")
    _check(lib.entmtp_verify_logits_stats(_p(hidden), _p(w_lm), T, hid, V, inv_temp, _p(logits),
                                          _p(entropy), _p(top1p), _p(argmax), _p(workspace),
                                          workspace.numel() * workspace.element_size(),
                                          _stream(stream)))


def stats_partials_bytes(T: int, hid: int, V: int) -> int:
    return int(lib.entmtp_stats_partials_bytes(T, hid, V))


def verify_logits_partials(hidden, w_lm, logits, inv_temp: float, partials, stream=None) -> None:
    """First half of verify_logits_stats: per-slice statistics partials, and
    the logits unless ``logits`` is None."""
    import torch
    _need(hidden.dim() == 2 and w_lm.dim() == 2, "hidden and w_lm are 2-D")
    T, hid = hidden.shape
    V = w_lm.shape[0]
    _dev(hidden, "hidden", torch.bfloat16, (T, hid))
    _dev(w_lm, "w_lm", torch.bfloat16, (V, hid))
    if logits is not None:
        _dev(logits, "logits", torch.float32, (T, V))
    _need(partials.is_cuda and partials.is_contiguous(), "partials must be a contiguous GPU tensor")
    _check(lib.entmtp_verify_logits_partials(_p(hidden), _p(w_lm), T, hid, V, inv_temp, _p(logits),
                                             _p(partials), partials.numel() * partials.element_size(),
                                             _stream(stream)))


def stats_finalize(partials, T: int, V: int, inv_temp: float, entropy, top1p, argmax,
                   stream=None) -> None:
    """Second half of verify_logits_stats: merges the partials into per-node statistics."""
    import torch
    _need(partials.is_cuda and partials.is_contiguous(), "partials must be a contiguous GPU tensor")
    for name, t, dt in (("entropy", entropy, torch.float32), ("top1p", top1p, torch.float32),
                        ("argmax", argmax, torch.int32)):
        if t is not None:
            _dev(t, name, dt, min_numel=T)
    _check(lib.entmtp_stats_finalize(_p(partials), T, V, inv_temp, _p(entropy), _p(top1p),
                                     _p(argmax), _stream(stream)))


def logit_stats(logits, inv_temp: float, entropy, top1p, argmax, stream=None) -> None:
    import torch
    _need(logits.dim() == 2, "logits are 2-D")
    T, V = logits.shape
    _dev(logits, "logits", torch.float32, (T, V))
    for name, t, dt in (("entropy", entropy, torch.float32), ("top1p", top1p, torch.float32),
                        ("argmax", argmax, torch.int32)):
        if t is not None:
            _dev(t, name, dt, min_numel=T)
    _check(lib.entmtp_logit_stats(_p(logits), T, V, inv_temp, _p(entropy), _p(top1p), _p(argmax),
                                  _stream(stream)))


def accept(bank: Bank, topo: int, draft_tokens, argmax, top1p, accept_len, path, bonus,
           best_top1p=None, stream=None) -> None:
    import torch
    _need(0 <= topo < len(bank), "topo out of range")
    T, D = bank.T[topo], bank.D[topo]
    _dev(draft_tokens, "draft_tokens", torch.int32, min_numel=T)
    _dev(argmax, "argmax", torch.int32, min_numel=T)
    if top1p is not None:
        _dev(top1p, "top1p", torch.float32, min_numel=T)
    _dev(accept_len, "accept_len", torch.int32, min_numel=1)
    _dev(path, "path", torch.int32, min_numel=D + 1)
    _dev(bonus, "bonus", torch.int32, min_numel=1)
    if best_top1p is not None:
        _dev(best_top1p, "best_top1p", torch.float32, min_numel=1)
    _check(lib.entmtp_accept(bank.handle, topo, _p(draft_tokens), _p(argmax), _p(top1p),
                             _p(accept_len), _p(path), _p(bonus), _p(best_top1p),
                             _stream(stream)))


def draft_logits(bank: Bank, topo: int, hidden, w_lm, draft_tokens, argmax, z_draft, z_top,
                 stream=None) -> None:
    import torch
    T = bank.T[topo]
    V, hid = w_lm.shape
    _dev(hidden, "hidden", torch.bfloat16, min_numel=T * hid)
    _need(hidden.shape[-1] == hid, "hidden rows have the LM head's width")
    _dev(w_lm, "w_lm", torch.bfloat16, (V, hid))
    _dev(draft_tokens, "draft_tokens", torch.int32, min_numel=T)
    _dev(argmax, "argmax", torch.int32, min_numel=T)
    _dev(z_draft, "z_draft", torch.float32, min_numel=T)
    _dev(z_top, "z_top", torch.float32, min_numel=T)
    _check(lib.entmtp_draft_logits(bank.handle, topo, _p(hidden), _p(w_lm), hid, V, _p(draft_tokens),
                                   _p(argmax), _p(z_draft), _p(z_top), _stream(stream)))


def accept_typical(bank: Bank, topo: int, draft_tokens, argmax, z_draft, z_top, entropy, top1p,
                   inv_temp: float, eps: float, alpha: float, accept_len, path, bonus,
                   best_top1p=None, stream=None) -> None:
    import torch
    T, D = bank.T[topo], bank.D[topo]
    for name, t, dt in (("draft_tokens", draft_tokens, torch.int32), ("argmax", argmax, torch.int32),
                        ("z_draft", z_draft, torch.float32), ("z_top", z_top, torch.float32),
                        ("entropy", entropy, torch.float32), ("top1p", top1p, torch.float32)):
        _dev(t, name, dt, min_numel=T)
    _dev(accept_len, "accept_len", torch.int32, min_numel=1)
    _dev(path, "path", torch.int32, min_numel=D + 1)
    _dev(bonus, "bonus", torch.int32, min_numel=1)
    _check(lib.entmtp_accept_typical(bank.handle, topo, _p(draft_tokens), _p(argmax), _p(z_draft),
                                     _p(z_top), _p(entropy), _p(top1p), inv_temp, eps, alpha,
                                     _p(accept_len), _p(path), _p(bonus), _p(best_top1p),
                                     _stream(stream)))


def frontier_tree(parent, max_depth: int):
    """The joint tree T u F of the offline search's scoring step
    (entmtp_frontier_tree): every node of T whose depth is below max_depth,
    the root included, proposes its next-ranked child; the candidates follow
    T's nodes in node order.  Returns (parent list of T u F, in_tree list of
    0/1)."""
    T = len(parent)
    _need(T >= 1, "the tree has a root")
    src = (_c_i32 * T)(*[int(p) for p in parent])
    cap = 2 * T
    joint = (_c_i32 * cap)()
    in_tree = (ctypes.c_uint8 * cap)()
    n = _c_i32(0)
    _check(lib.entmtp_frontier_tree(src, T, int(max_depth), joint, in_tree, cap, ctypes.byref(n)))
    return list(joint[: n.value]), list(in_tree[: n.value])


def frontier_score(bank: Bank, topo: int, in_tree, sums, best, local_ok=None, draft_tokens=None,
                   argmax=None, stream=None) -> None:
    """Scores of T's one-node augmentations from samples of the joint tree
    (bank tree ``topo``): local_ok uint8 [S, T], or draft_tokens and argmax
    int32 [S, T] for the greedy test."""
    import torch
    T = bank.T[topo]
    _dev(in_tree, "in_tree", torch.uint8, min_numel=T)
    _dev(sums, "sums", torch.int32, min_numel=T)
    _dev(best, "best", torch.int32, min_numel=1)
    if local_ok is not None:
        _dev(local_ok, "local_ok", torch.uint8)
        _need(local_ok.dim() == 2 and local_ok.shape[1] == T, "local_ok is [S, T]")
        S = local_ok.shape[0]
    else:
        _need(draft_tokens is not None and argmax is not None,
              "give local_ok, or draft_tokens and argmax")
        _dev(draft_tokens, "draft_tokens", torch.int32)
        _dev(argmax, "argmax", torch.int32)
        _need(draft_tokens.dim() == 2 and draft_tokens.shape[1] == T and
              argmax.shape == draft_tokens.shape, "draft_tokens and argmax are [S, T]")
        S = draft_tokens.shape[0]
    _check(lib.entmtp_frontier_score(bank.handle, topo, _p(in_tree), S, _p(local_ok),
                                     _p(draft_tokens), _p(argmax), _p(sums), _p(best),
                                     _stream(stream)))


def accept_stochastic(bank: Bank, topo: int, draft_tokens, logits, q, inv_temp: float, argmax,
                      top1p, u_accept, u_sample, workspace, accept_len, path, bonus,
                      stream=None) -> None:
    """Speculative-sampling tree verification; logits and q fp32 [T, V],
    argmax / top1p the logits' statistics at inv_temp, uniforms fp32 [T],
    workspace fp32 [V]."""
    import torch
    T, D = bank.T[topo], bank.D[topo]
    _need(logits.dim() == 2 and logits.shape[0] >= T, "logits is [T, V]")
    V = logits.shape[1]
    _dev(logits, "logits", torch.float32)
    _dev(q, "q", torch.float32, tuple(logits.shape))
    _dev(draft_tokens, "draft_tokens", torch.int32, min_numel=T)
    _dev(argmax, "argmax", torch.int32, min_numel=T)
    _dev(top1p, "top1p", torch.float32, min_numel=T)
    _dev(u_accept, "u_accept", torch.float32, min_numel=T)
    _dev(u_sample, "u_sample", torch.float32, min_numel=T)
    _dev(workspace, "workspace", torch.float32, min_numel=V)
    _dev(accept_len, "accept_len", torch.int32, min_numel=1)
    _dev(path, "path", torch.int32, min_numel=D + 1)
    _dev(bonus, "bonus", torch.int32, min_numel=1)
    _check(lib.entmtp_accept_stochastic(bank.handle, topo, _p(draft_tokens), _p(logits), _p(q), V,
                                        inv_temp, _p(argmax), _p(top1p), _p(u_accept),
                                        _p(u_sample), _p(workspace),
                                        _p(accept_len), _p(path), _p(bonus), _stream(stream)))


def kv_compact(path, accept_len, prefix_len: int, k_cache, v_cache, stream=None) -> None:
    """Caches [Hkv,cap,d] (one layer) or [n_layers,Hkv,cap,d] (bf16)."""
    import torch
    _need(k_cache.dim() in (3, 4) and v_cache.shape == k_cache.shape, "caches are 3-D or 4-D, equal shapes")
    _dev(k_cache, "k_cache", torch.bfloat16)
    _dev(v_cache, "v_cache", torch.bfloat16)
    _dev(path, "path", torch.int32, min_numel=1)
    _dev(accept_len, "accept_len", torch.int32, min_numel=1)
    if k_cache.dim() == 3:
        n_layers, (Hkv, cap, d) = 1, k_cache.shape
        stride = Hkv * cap * d
    else:
        n_layers, Hkv, cap, d = k_cache.shape
        stride = Hkv * cap * d
    _check(lib.entmtp_kv_compact(_p(path), path.numel(), _p(accept_len), prefix_len, _p(k_cache),
                                 _p(v_cache), n_layers, stride, Hkv, cap, d, _stream(stream)))


def ladder_next(rung: int, n_rungs: int, s: float, tau_on: float, tau_off: float) -> int:
    return _check(lib.entmtp_ladder_next(rung, n_rungs, s, tau_on, tau_off))


def ladder_next_batched(rung: np.ndarray, s: np.ndarray, n_rungs: int, tau_on: float,
                        tau_off: float) -> None:
    """rung: int32 host array [B], moved in place on float32 s [B]."""
    _need(isinstance(rung, np.ndarray) and rung.dtype == np.int32 and rung.flags.c_contiguous,
          "rung must be a contiguous int32 numpy array")
    _need(isinstance(s, np.ndarray) and s.dtype == np.float32 and s.flags.c_contiguous
          and s.shape == rung.shape, "s must be a contiguous float32 numpy array shaped like rung")
    _check(lib.entmtp_ladder_next_batched(rung.size, _np_p(rung), _np_p(s), n_rungs, tau_on,
                                          tau_off))


def version() -> str:
    return lib.entmtp_version().decode()


# --------------------------------------------------------------------- step --

class Step:
    """A verification-step context (entmtp_step_*): the caches, the LM head and
    the per-step outputs are fixed at construction; ``launch`` enqueues one
    step and ``wait`` returns (accept_len, bonus, best_top1p) from the host
    record the acceptance kernel publishes.  Output tensors are allocated here
    and exposed as attributes (logits, entropy, top1p, argmax, accept_len,
    bonus, best_top1p, path)."""

    def __init__(self, bank: Bank, k_cache, v_cache, w_lm, *, n_layers=1, Hq, Hkv, d=HEAD_DIM,
                 cap, tree_rows, scale, rope_theta, inv_temp=1.0, cache_layer_stride=0,
                 keep_logits=True, tau_on=0.8, tau_off=0.6, device_prefix_fixed=False,
                 stream=None):
        import torch
        dev = k_cache.device
        V, hid = w_lm.shape
        D = max(bank.D)
        self.logits = (torch.empty((tree_rows, V), dtype=torch.float32, device=dev) if keep_logits
                       else None)
        # zeroed: a step writes rows [0, T) only, and rows above stay defined
        self.entropy = torch.zeros(tree_rows, dtype=torch.float32, device=dev)
        self.top1p = torch.zeros(tree_rows, dtype=torch.float32, device=dev)
        self.argmax = torch.zeros(tree_rows, dtype=torch.int32, device=dev)
        self.accept_len = torch.zeros(1, dtype=torch.int32, device=dev)
        self.bonus = torch.zeros(1, dtype=torch.int32, device=dev)
        self.best_top1p = torch.zeros(1, dtype=torch.float32, device=dev)
        self.path = torch.full((D + 1,), -1, dtype=torch.int32, device=dev)
        _dev(k_cache, "k_cache", torch.bfloat16)
        _dev(v_cache, "v_cache", torch.bfloat16)
        _dev(w_lm, "w_lm", torch.bfloat16, (V, hid))
        self._keep = (bank, k_cache, v_cache, w_lm)
        c = StepConfig(n_layers, Hq, Hkv, d, cap, tree_rows, scale, rope_theta,
                       k_cache.data_ptr(), v_cache.data_ptr(), cache_layer_stride, w_lm.data_ptr(),
                       hid, V, inv_temp, None if self.logits is None else self.logits.data_ptr(),
                       self.entropy.data_ptr(),
                       self.top1p.data_ptr(), self.argmax.data_ptr(), self.accept_len.data_ptr(),
                       self.bonus.data_ptr(), self.best_top1p.data_ptr(), self.path.data_ptr(),
                       D + 1, None, 0, _stream(stream).value, tau_on, tau_off,
                       int(bool(device_prefix_fixed)))
        need = int(lib.entmtp_step_workspace(bank.handle, ctypes.byref(c)))
        if need == 0:
            _check(lib.entmtp_step_create(bank.handle, ctypes.byref(c), ctypes.byref(_c_p())))
            raise EntmtpError(EINVAL, "invalid step configuration")
        self.workspace = torch.empty(need + 256, dtype=torch.uint8, device=dev)
        base = self.workspace.data_ptr()
        c.workspace = (base + 255) // 256 * 256
        c.workspace_bytes = need
        self.config = c
        h = _c_p()
        _check(lib.entmtp_step_create(bank.handle, ctypes.byref(c), ctypes.byref(h)))
        self._h = h
        self._a, self._b, self._s = _c_i32(), _c_i32(), _c_f32()

    @property
    def handle(self):
        return self._h

    def launch(self, topo: int, prefix_len: int, q, k_tree, v_tree, out, hidden, draft_tokens,
               ev_lm_begin=None, ev_lm_end=None, w_lm=None) -> None:
        """One host-scheduled step; the previous step's compaction goes with it
        (``flush`` completes the cache on the configured stream)."""
        ev = [None if e is None else _c_p(e.cuda_event) for e in (ev_lm_begin, ev_lm_end)]
        _check(lib.entmtp_step_launch(self._h, topo, prefix_len, _p(q), _p(k_tree), _p(v_tree),
                                      _p(out), _p(hidden), _p(w_lm), _p(draft_tokens), ev[0],
                                      ev[1]))

    def arm(self, hidden, T_bound: int, w_lm=None, ev_lm_begin=None, ev_lm_end=None) -> None:
        """Enqueue the next step's LM head (rows [0, T_bound) of ``hidden``)
        behind a gate that the next ``launch`` opens."""
        ev = [None if e is None else _c_p(e.cuda_event) for e in (ev_lm_begin, ev_lm_end)]
        _check(lib.entmtp_step_arm(self._h, _p(hidden), _p(w_lm), T_bound, ev[0], ev[1]))

    def flush(self) -> None:
        _check(lib.entmtp_step_flush(self._h))

    def wait(self, timeout_s: float = 30.0):
        _check(lib.entmtp_step_wait(self._h, ctypes.byref(self._a), ctypes.byref(self._b),
                                    ctypes.byref(self._s), timeout_s))
        return self._a.value, self._b.value, self._s.value

    def device_start(self, topo: int, prefix_len: int) -> None:
        _check(lib.entmtp_step_device_start(self._h, topo, prefix_len))

    def launch_device(self, q, k_tree, v_tree, out, hidden, drafts, log=None, w_lm=None,
                      ev_lm_begin=None, ev_lm_end=None) -> None:
        """One device-scheduled step; drafts [K, tree_rows] int32; log int32 [rows, 4]
        (row = device step count % rows) or None."""
        ev = [None if e is None else _c_p(e.cuda_event) for e in (ev_lm_begin, ev_lm_end)]
        rows = 0 if log is None else log.numel() // 4
        _check(lib.entmtp_step_launch_device(self._h, _p(q), _p(k_tree), _p(v_tree), _p(out),
                                             _p(hidden), _p(w_lm), _p(drafts), _p(log), rows,
                                             ev[0], ev[1]))

    def device_graph(self, steps, log=None):
        """Capture device-scheduled steps as one replayable graph: ``steps`` is a
        list (length a multiple of 4) of dicts with q, k_tree, v_tree, out,
        hidden, drafts and optionally w_lm.  Returns a StepGraph."""
        n = len(steps)
        arr = lambda key: _host_ptrs([e.get(key) for e in steps])   # noqa: E731
        h = _c_p()
        rows = 0 if log is None else log.numel() // 4
        w = arr("w_lm") if any(e.get("w_lm") is not None for e in steps) else None
        _check(lib.entmtp_step_device_graph(self._h, n, arr("q"), arr("k_tree"), arr("v_tree"),
                                            arr("out"), arr("hidden"), w, arr("drafts"), _p(log),
                                            rows, ctypes.byref(h)))
        return StepGraph(self, h, steps, log)

    def close(self):
        if getattr(self, "_h", None):
            lib.entmtp_step_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class StepGraph:
    """A captured segment of device-scheduled steps (entmtp_step_device_graph);
    keeps the tensors it was captured with alive."""

    def __init__(self, step: Step, handle, keep, log):
        self._step, self._h, self._keep = step, handle, (keep, log)

    def launch(self) -> None:
        _check(lib.entmtp_step_graph_launch(self._step.handle, self._h))

    def close(self):
        if getattr(self, "_h", None):
            lib.entmtp_step_graph_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
