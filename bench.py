#!/usr/bin/env python3
"""Tree-verification step benchmark on one MI355X.

A step is one pass of the whole verification hot path at batch 1:
  pick the tree for this step (the hysteretic ladder, tau_on 0.8, tau_off 0.6,
        over the previous step's top-1 probability at the deepest accepted
        node; a one-tree bank always picks its tree);
  GPU:  tree attention (tree K/V appended to the cache), LM-head logits with
        fused softmax statistics -> greedy acceptance, and KV compaction (the
        compaction of a step goes out with the next step's launch, on the
        cache stream, beside the next LM head).
The ladder runs either on the GPU, in the acceptance kernel, which leaves the
next step's tree and prefix in device memory (device-scheduled steps: the
host enqueues step after step and reads nothing back), or on the host, which
polls the pinned record acceptance publishes (accept length, s, path) -- the
step's one device-to-host read -- moves the prefix and launches the next step
(whose LM head it enqueued ahead, behind a gate).  The default workload runs
device-scheduled and reports the host-scheduled loop beside it.
The timed region ends with a flush, so it holds exactly K compactions.

Default workload: Vicuna-7B shapes (32 x 128 heads, hidden 4096, vocabulary
32000), one attention layer and the LM head, a 27-node tree of depth 4 over
a 256-token prefix, the prefix reset every step (each step verifies a fresh
tree at the same position).  ``--workload`` selects the others: the 5-tree
bank {1, 8, 26, 64, 128} at prefix 2048 growing every step, the 32-layer
stack, the 13B shapes and the batch-8 GQA step.  Inputs are seeded synthetic
tensors staged in HBM before timing (a pool of per-step inputs is cycled);
two copies of the LM-head weight alternate between steps so that the 256 MB
last-level cache cannot serve the weight stream.

After the default run, a switching study on the 5-tree bank (prefix fixed at
2048) compares steps whose tree the ladder picks, and steps whose tree moves
by one rung every step, with steps on one fixed tree each, weighted by the
same tree-size histogram; arming is the same in all runs, so the difference
is what switching trees costs.

Prints ONE JSON line.  ``--gpus N`` with N > 1 exits: the build targets one GPU.
"""
from __future__ import annotations

import argparse
import ctypes
import gc
import json
import math
import os
import sys
import time

import numpy as np

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
METRIC = "tree-verify steps/sec and µs/step at batch 1; achieved HBM GB/s vs peak"
MIN_TIMED_LAUNCHES = 16
SINGLE_WORKLOADS = ["tree27_L256_7b", "bank5_L2048_7b", "tree64_L4096_7b_32layer",
                    "tree128_L8192_13b"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="tree27_L256_7b",
                    choices=SINGLE_WORKLOADS + ["batch8_gqa_v128k"])
    ap.add_argument("--pool", type=int, default=32, help="distinct per-step input sets")
    ap.add_argument("--weight-copies", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the switching study and the timings of the typical-acceptance, "
                         "speculative-sampling and frontier kernels")
    ap.add_argument("--event-every", type=int, default=8,
                    help="time the LM head with HIP events on a seeded random 1/n of the timed steps "
                         f"(at least {MIN_TIMED_LAUNCHES}; each event pair costs the host a few "
                         "microseconds)")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0)
    ap.add_argument("--switch-steps", type=int, default=300,
                    help="timed steps per run of the switching study")
    ap.add_argument("--fixed-topo", type=int, default=-1,
                    help="disable the scheduler and use this bank entry every step")
    ap.add_argument("--graph", action="store_true",
                    help="with --gpu-scheduler: replay segments of steps captured as HIP graphs")
    ap.add_argument("--no-arm", action="store_true",
                    help="host-scheduled steps: launch each LM head only after the previous "
                         "result is read, instead of enqueueing it ahead behind a gate")
    ap.add_argument("--scheduler", choices=["auto", "gpu", "host"], default="auto",
                    help="where the ladder runs: on the GPU (no result read per step, the next "
                         "step's tree and prefix stay in device memory) or on the host (one "
                         "record read per step); auto: the GPU for the 27-node workload, whose "
                         "timed loop is then followed by a host-scheduled run reported beside "
                         "it, the host for the others")
    ap.add_argument("--gpu-scheduler", action="store_true", help="same as --scheduler gpu")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run plain 256 MiB device copies (reference for HBM byte counters)")
    ap.add_argument("--lm-rows", default="",
                    help="only time the LM head with statistics partials over this many rows "
                         "(comma-separated counts; the batched verification pass's many-row "
                         "case), one JSON line per count")
    ap.add_argument("--lm-vocab", type=int, default=128256)
    ap.add_argument("--lm-hidden", type=int, default=4096)
    ap.add_argument("--lm-calls", type=int, default=30)
    return ap.parse_args()


def calibrate_copy():
    """Plain device-to-device copies of a known size: the reference that scales
    the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    n = 256 << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read_per_copy": n,
                      "bytes_written_per_copy": n, "copies": 5}))


class TimingEvent:
    """A HIP timing event without the system-scope fence at record time
    (hipEventDisableSystemFence): the bracketed kernel's results stay on the
    device, and the fence would add its cache write-back to the bracket.
    Created through the HIP runtime torch loaded."""
    _hip = None

    def __init__(self):
        if TimingEvent._hip is None:
            with open("/proc/self/maps") as f:
                rt = sorted({l.split()[-1] for l in f if "libamdhip64" in l})
            hip = ctypes.CDLL(rt[0])
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
            hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
            TimingEvent._hip = hip
        self.ptr = ctypes.c_void_p()
        rc = TimingEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.ptr), 0x20000000)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def elapsed_time(self, end) -> float:
        ms = ctypes.c_float()
        rc = TimingEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.ptr, end.ptr)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def __del__(self):
        if self._hip is not None and self.ptr:
            self._hip.hipEventDestroy(self.ptr)


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def lm_rows(args, api, torch):
    """The LM head with statistics partials (entmtp_verify_logits_partials,
    no logits) over T rows, for each requested T: `--lm-calls` back-to-back
    calls between two events after five untimed ones; seeded N(0, 1) hidden
    rows, W ~ N(0, 0.02^2), bf16."""
    V, hid = args.lm_vocab, args.lm_hidden
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(11)
    W = (torch.randn((V, hid), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    for T in (int(x) for x in args.lm_rows.split(",") if x):
        X = torch.randn((T, hid), generator=g, device=dev).to(torch.bfloat16)
        ws = torch.empty(api.stats_partials_bytes(T, hid, V), dtype=torch.uint8, device=dev)
        for _ in range(5):
            api.verify_logits_partials(X, W, None, 1.0, ws)
        torch.cuda.synchronize()
        e0, e1 = TimingEvent(), TimingEvent()
        hip = TimingEvent._hip
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        hip.hipEventRecord(e0.ptr, stream)
        for _ in range(args.lm_calls):
            api.verify_logits_partials(X, W, None, 1.0, ws)
        hip.hipEventRecord(e1.ptr, stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.lm_calls
        flops = 2.0 * T * V * hid
        print(json.dumps({"lm_head_rows": T, "vocab": V, "hidden": hid, "calls": args.lm_calls,
                          "us_per_call": round(us, 2),
                          "TFLOPs": round(flops / us / 1e6, 1),
                          "mfma_frac_bf16": round(flops / us / 1e6 / MFMA_PEAK_BF16_TFLOPS, 4),
                          "W_GBps": round(V * hid * 2 / us / 1e3, 1),
                          "timing": "HIP events around back-to-back calls on one stream"}),
              flush=True)


class SingleSeq:
    """A single-sequence workload staged in HBM: the LM-head weight copies, the
    per-layer caches, a pool of per-step inputs with their draft tokens for
    every bank tree, and one step context on a stream of its own."""

    def __init__(self, api, synth, torch, name, pool_size, weight_copies, cap_steps,
                 device_prefix_fixed=False):
        self.api, self.synth, self.torch, self.lib = api, synth, torch, api.lib
        dev = self.dev = torch.device("cuda:0")
        wl = self.wl = synth.WORKLOADS[name]
        self.Hq, self.Hkv, self.d, self.hid, self.V = (wl.n_heads, wl.n_kv_heads, wl.head_dim,
                                                       wl.hidden, wl.vocab)
        Hq, Hkv, d, hid, V = self.Hq, self.Hkv, self.d, self.hid, self.V
        self.trees = synth.workload_trees(wl)
        self.bank = api.Bank(self.trees)
        self.n_topo = len(self.trees)
        self.Ts = self.bank.T
        Tmax, Dmax = max(self.bank.T), max(self.bank.D)
        self.L0 = wl.prefix_len
        self.cap = cap = self.L0 + cap_steps * (Dmax + 1) + Tmax + 64
        self.scale, self.theta = 1.0 / math.sqrt(d), wl.rope_theta
        self.NL = NL = wl.n_layers
        log(f"workload {wl.name}: bank T={self.bank.T} D={self.bank.D}, L0={self.L0}, cap={cap}")
        t0 = time.time()
        bf = torch.bfloat16

        def to_dev(bits):
            return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(bf).to(dev)

        self.w_host = synth.lm_head_weight(wl.ident, V, hid)
        W = [to_dev(self.w_host)]
        for _ in range(1, weight_copies):
            W.append(W[0].clone())
        self.W = W
        base = synth.attn_inputs(wl.ident, 1, Hq, Hkv, d, self.L0, cap)
        self.kc0_host = base.k_cache[:, :self.L0].copy()
        self.vc0_host = base.v_cache[:, :self.L0].copy()
        self.k_cache = torch.zeros((NL, Hkv, cap, d), dtype=bf, device=dev)   # [layer][head][slot][dim]
        self.v_cache = torch.zeros((NL, Hkv, cap, d), dtype=bf, device=dev)
        self.k_cache[0, :, :self.L0] = to_dev(self.kc0_host)
        self.v_cache[0, :, :self.L0] = to_dev(self.vc0_host)
        del base
        # further layers (the 32-layer workload): seeded N(0, 1) drawn on the
        # GPU, a generator per layer (the oracle baseline covers one layer)
        gen = torch.Generator(device=dev)

        def randn_dev(shape, seed):
            gen.manual_seed(seed)
            return torch.randn(shape, generator=gen, device=dev, dtype=torch.float32).to(bf)

        for l in range(1, NL):
            self.k_cache[l, :, :self.L0] = randn_dev((Hkv, self.L0, d), 1000 * wl.ident + 2 * l)
            self.v_cache[l, :, :self.L0] = randn_dev((Hkv, self.L0, d), 1000 * wl.ident + 2 * l + 1)

        # the scheduler workload plants a confidence regime in the hidden
        # states (a lift on one token per row) so that the ladder moves
        lifted = self.n_topo > 1
        P = self.P = pool_size if NL == 1 else min(pool_size, 4)
        deltas, spike_tok = synth.regime_spikes(wl.ident, P, Tmax, V, hid)
        pool = []
        for e in range(P):
            a_in = synth.attn_inputs(wl.ident, Tmax, Hq, Hkv, d, 0, Tmax, step=e + 1)
            x = synth.hidden_rows(wl.ident, Tmax, hid, step=e + 1)
            if lifted:
                x = synth.plant_spike(x, self.w_host, spike_tok[e], float(deltas[e]), wl.w_std)
            u, r = synth.draft_randoms(wl.ident, Tmax, V, step=e + 1)
            q_l, kt_l, vt_l = [to_dev(a_in.q)], [to_dev(a_in.k_tree)], [to_dev(a_in.v_tree)]
            for l in range(1, NL):   # layer-major, as the step reads them
                sd = 1000 * wl.ident + 100 * (e + 1) + 3 * l
                q_l.append(randn_dev((Tmax, Hq, d), sd))
                kt_l.append(randn_dev((Tmax, Hkv, d), sd + 1))
                vt_l.append(randn_dev((Tmax, Hkv, d), sd + 2))
            pool.append({"q": torch.stack(q_l), "kt": torch.stack(kt_l), "vt": torch.stack(vt_l),
                         "x": to_dev(x), "u": u, "r": r,
                         "host": (a_in.q, a_in.k_tree, a_in.v_tree, x)})
        self.pool = pool
        log(f"staged inputs in {time.time() - t0:.1f}s")

        # the step loop runs on a stream of its own (non-blocking: launches on
        # the legacy default stream cost the host more); the LM-head weight
        # copy is passed per step; the statistics come from the LM head's
        # accumulators, so no logits are materialised
        self.stream = torch.cuda.Stream()
        self.st = api.Step(self.bank, self.k_cache, self.v_cache, W[0], n_layers=NL, Hq=Hq,
                           Hkv=Hkv, d=d, cap=cap, tree_rows=Tmax, scale=self.scale,
                           rope_theta=self.theta, keep_logits=False, tau_on=0.8, tau_off=0.6,
                           device_prefix_fixed=device_prefix_fixed,
                           cache_layer_stride=Hkv * cap * d, stream=self.stream)
        torch.cuda.synchronize()
        self.out = torch.empty((NL, Tmax, Hq, d), dtype=bf, device=dev)

        # draft tokens: the target's greedy token at the parent with
        # probability p_acc, computed with the library itself on each pool
        # entry (input synthesis; the separate logits and statistics kernels,
        # so that the counters of the timed fused kernel are not mixed with
        # these staging launches)
        lg = torch.empty((Tmax, V), dtype=torch.float32, device=dev)
        for e in pool:
            api.verify_logits(e["x"], W[0], lg)
            api.logit_stats(lg, 1.0, None, None, self.st.argmax)
            am = self.st.argmax.cpu().numpy()
            e["tok"] = [synth.draft_tokens(self.trees[k], am, e["u"], e["r"], wl.p_acc)
                        for k in range(self.n_topo)]
            e["tok_dev"] = [torch.from_numpy(t).to(dev) for t in e["tok"]]
            table = np.zeros((self.n_topo, Tmax), np.int32)
            for k, t in enumerate(e["tok"]):
                table[k, : len(t)] = t
            e["drafts_dev"] = torch.from_numpy(table).to(dev)
        del lg
        torch.cuda.synchronize()
        P_ = ctypes.c_void_p
        self.pool_p = [{"q": P_(e["q"].data_ptr()), "kt": P_(e["kt"].data_ptr()),
                        "vt": P_(e["vt"].data_ptr()), "x": P_(e["x"].data_ptr()),
                        "tok": [P_(t.data_ptr()) for t in e["tok_dev"]],
                        "drafts": P_(e["drafts_dev"].data_ptr())} for e in pool]
        self.W_p = [P_(w.data_ptr()) for w in W]
        self.out_p = P_(self.out.data_ptr())

    def chk(self, rc):
        if rc:
            raise self.api.EntmtpError(rc, self.api.last_error())

    def run(self, K, warmup, policy, *, grow, start_rung=0, arm=True, arm_reach=True,
            n_events=0, event_pass=0, on_gpu=False, graph=False, step_times=None):
        """Runs `warmup` untimed and K timed steps.  policy(topo, s) gives the
        next step's tree from the current one and the step's s (host-
        scheduled steps).  grow: the prefix grows by the accepted tokens (else
        every step verifies at L0).  arm: each next step's LM head is enqueued
        behind a gate while the step before is pending, sized for the next
        rung (arm_reach) or for the current tree.  n_events: timed steps whose
        LM head carries a HIP event pair (a seeded random choice);
        event_pass: steps run right after the timed region (same loop, inputs
        and state, outside the timing) whose LM heads all carry event pairs.  on_gpu:
        the ladder runs on the GPU (entmtp_step_launch_device), optionally
        replayed as captured graph segments (the prefix then grows unless the
        step context was made with a fixed device prefix).  step_times: a list
        that receives the host clock after every timed step."""
        torch, lib = self.torch, self.lib
        h = self.st.handle
        Ts, n_topo, P = self.Ts, self.n_topo, self.P
        pool_p, W_p, out_p = self.pool_p, self.W_p, self.out_p
        total = warmup + K + event_pass
        steplog = torch.full((total, 4), -1, dtype=torch.int32, device=self.dev)
        log_base = ctypes.c_void_p(steplog.data_ptr())
        a_c, b_c, s_c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_float()
        a_r, b_r, s_r = ctypes.byref(a_c), ctypes.byref(b_c), ctypes.byref(s_c)
        state = {"L": self.L0, "rung": start_rung}
        armed = [False, 0]        # armed?, the rows the armed LM head covers
        lm_rows = []              # rows of the LM head each host-scheduled step ran
        chk = self.chk

        def step_gpu(t, ev=(None, None)):
            # nothing is read back: the next step's tree and prefix stay on the GPU
            e = pool_p[t % P]
            chk(lib.entmtp_step_launch_device(h, e["q"], e["kt"], e["vt"], out_p, e["x"],
                                              W_p[t % len(W_p)], e["drafts"], log_base, total,
                                              ev[0], ev[1]))

        def step(t, ev=(None, None), ev_next=(None, None), arm_next=False):
            L = state["L"] if grow else self.L0
            topo = state["rung"]
            e = pool_p[t % P]
            if armed[0]:   # the LM head and its events are in the queue already
                ev = (None, None)
            chk(lib.entmtp_step_launch(h, topo, L, e["q"], e["kt"], e["vt"], out_p, e["x"],
                                       W_p[t % len(W_p)], e["tok"][topo], ev[0], ev[1]))
            lm_rows.append(armed[1] if armed[0] and Ts[topo] <= armed[1] else Ts[topo])
            armed[0] = False
            if arm and arm_next:
                nx = pool_p[(t + 1) % P]
                bound = Ts[min(topo + 1, n_topo - 1)] if arm_reach else Ts[topo]
                chk(lib.entmtp_step_arm(h, nx["x"], W_p[(t + 1) % len(W_p)], bound, ev_next[0],
                                        ev_next[1]))
                armed[:] = [True, bound]
            chk(lib.entmtp_step_wait(h, a_r, b_r, s_r, 30.0))
            a, s = a_c.value, s_c.value
            if grow:
                state["L"] = L + a + 1
            state["rung"] = policy(topo, s)
            return Ts[topo], L, a, s, topo

        # timed steps whose LM head carries an event pair: a seeded random
        # choice (a fixed stride can alias with the ladder's cycle through the
        # bank)
        sampled = sorted(np.random.default_rng(7).choice(K, min(K, n_events), replace=False).tolist())
        events = [(TimingEvent(), TimingEvent()) for _ in sampled]
        ev_p = {t: (a_.ptr, b_.ptr) for t, (a_, b_) in zip(sampled, events)}
        trace = []
        graphs, graph_steps = [], 0
        if on_gpu:
            chk(lib.entmtp_step_device_start(h, state["rung"], self.L0))
        torch.cuda.synchronize()
        # no garbage collection inside the timed region: a full collection of
        # the interpreter's heap stalls the host loop for tens of milliseconds
        # (collected before the warm-up, so that the warm-up steps run right
        # before the timed ones and the GPU does not sit idle in between)
        gc.collect()
        gc.disable()
        for t in range(warmup):
            if on_gpu:
                step_gpu(t)
            else:
                step(t, arm_next=t + 1 < warmup)
        chk(lib.entmtp_step_flush(h))   # the last warm-up step's compaction
        if on_gpu and graph:
            # segments of SEG steps (a whole number of input-pool and
            # weight-copy cycles, and of the 16-slot device state ring), all captured
            # after the warm-up, before the timed region; the steps past the last whole segment
            # run eagerly (and carry the LM-head events, which graph replays
            # do not)
            SEG = math.lcm(P, len(W_p), 16)
            for g0 in range(0, K - K % SEG, SEG):
                ts = range(warmup + g0, warmup + g0 + SEG)
                arr = lambda vals: (ctypes.c_void_p * SEG)(*[v.value for v in vals])   # noqa: E731
                gh = ctypes.c_void_p()
                chk(lib.entmtp_step_device_graph(
                    h, SEG, arr([pool_p[t % P]["q"] for t in ts]),
                    arr([pool_p[t % P]["kt"] for t in ts]), arr([pool_p[t % P]["vt"] for t in ts]),
                    arr([out_p] * SEG), arr([pool_p[t % P]["x"] for t in ts]),
                    arr([W_p[t % len(W_p)] for t in ts]), arr([pool_p[t % P]["drafts"] for t in ts]),
                    log_base, total, ctypes.byref(gh)))
                graphs.append(gh)
            graph_steps = len(graphs) * SEG
            sampled = [t for t in sampled if t >= graph_steps]
            log(f"captured {len(graphs)} graphs of {SEG} steps")
        torch.cuda.synchronize()
        # HIP API calls between two hipMemGetInfo calls are the timed region's
        # (the marker a rocprofv3 API trace of this run is cut at)
        torch.cuda.mem_get_info()
        t_start = time.perf_counter()
        for g in graphs:
            chk(lib.entmtp_step_graph_launch(h, g))
        for t in range(graph_steps, K):
            if on_gpu:
                step_gpu(warmup + t, ev_p.get(t, (None, None)))
            else:
                trace.append(step(warmup + t, ev_p.get(t, (None, None)),
                                  ev_p.get(t + 1, (None, None)), t + 1 < K))
            if step_times is not None:
                step_times.append(time.perf_counter())
        chk(lib.entmtp_step_flush(h))   # the last timed step's compaction
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
        torch.cuda.mem_get_info()
        if step_times is not None:
            step_times.insert(0, t_start)
        events = [ev for t, ev in zip(ev_p, events) if t >= graph_steps]
        for g in graphs:
            lib.entmtp_step_graph_destroy(g)
        n_timed_rows = len(lm_rows)
        # the event pass: every LM head bracketed, outside the timed region
        pass_events = [(TimingEvent(), TimingEvent()) for _ in range(event_pass)]
        pass_trace = []
        for j in range(event_pass):
            t = warmup + K + j
            ev = (pass_events[j][0].ptr, pass_events[j][1].ptr)
            if on_gpu:
                step_gpu(t, ev)
            else:
                nxt = (pass_events[j + 1][0].ptr, pass_events[j + 1][1].ptr) if j + 1 < event_pass \
                    else (None, None)
                pass_trace.append(step(t, ev, nxt, j + 1 < event_pass))
        if event_pass:
            chk(lib.entmtp_step_flush(h))
            torch.cuda.synchronize()
        gc.enable()
        if on_gpu:   # the steps' (tree, prefix, accept length, s) as the GPU logged them
            lg = steplog.cpu().numpy()
            rows = [(Ts[int(r)], int(L), int(a), float(np.int32(sb).view(np.float32)), int(r))
                    for r, L, a, sb in lg]
            trace = rows[warmup:warmup + K]
            pass_trace = rows[warmup + K:]
            state["L"] = int(lg[warmup + K - 1, 1] + lg[warmup + K - 1, 2] + 1)
        lm_ms = [a.elapsed_time(b) for a, b in events]
        pass_ms = [a.elapsed_time(b) for a, b in pass_events]
        timed_rows = lm_rows[n_timed_rows - len(trace):n_timed_rows] if n_timed_rows >= len(trace) else []
        return {"elapsed": elapsed, "trace": trace, "lm_ms": lm_ms, "sampled": sampled,
                "lm_rows": timed_rows, "L_end": state["L"], "pass_ms": pass_ms,
                "pass_T": [T for T, *_ in pass_trace]}


def ladder(lib, n_topo):
    return lambda topo, s: lib.entmtp_ladder_next(topo, n_topo, s, 0.8, 0.6)


def histogram(vals):
    h = {}
    for v in vals:
        h[v] = h.get(v, 0) + 1
    return dict(sorted(h.items()))


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the tree-verification path is single-GPU "
              "(sharding across GPUs -- KV heads and vocabulary slices -- is designed, not built)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_27550_amd import api, synth

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.lm_rows:
        lm_rows(args, api, torch)
        return
    torch.cuda.set_device(torch.device("cuda:0"))
    lib = api.lib

    if args.workload == "batch8_gqa_v128k":
        run_batched(args, api, synth, torch, lib)
        return
    grows = args.workload == "bank5_L2048_7b"
    total_steps = args.warmup + args.steps
    run = SingleSeq(api, synth, torch, args.workload, args.pool, args.weight_copies,
                    total_steps if grows else 0, device_prefix_fixed=not grows)
    wl, bank = run.wl, run.bank
    Hq, Hkv, d, hid, V, NL = run.Hq, run.Hkv, run.d, run.hid, run.V, run.NL
    sched = "gpu" if args.gpu_scheduler else args.scheduler
    if sched == "auto":
        sched = "gpu" if args.workload == "tree27_L256_7b" else "host"
    on_gpu = sched == "gpu"
    fixed = args.fixed_topo >= 0
    policy = (lambda topo, s: args.fixed_topo) if fixed else ladder(lib, run.n_topo)
    K = args.steps
    n_events = max(1, K // max(1, args.event_every))
    res = run.run(K, args.warmup, policy, grow=grows, start_rung=max(args.fixed_topo, 0),
                  arm=not args.no_arm, arm_reach=not fixed, n_events=n_events,
                  event_pass=MIN_TIMED_LAUNCHES, on_gpu=on_gpu, graph=args.graph)
    elapsed, trace = res["elapsed"], res["trace"]
    sampled = [t for t in res["sampled"]]
    # LM-head durations: the timed region's sample, then the event pass
    lm_T = [trace[t][0] for t in sampled][:len(res["lm_ms"])] + res["pass_T"]
    lm_ms = res["lm_ms"] + res["pass_ms"]
    n_in_region = len(res["lm_ms"])
    by_T = {}
    for T, ms in zip(lm_T, lm_ms):
        by_T.setdefault(T, []).append(ms)
    lm_us_by_T = {str(T): round(float(np.mean(v)) * 1e3, 2) for T, v in sorted(by_T.items())}

    # algorithmic bytes (what the method must move; fp32 logits excluded)
    def step_bytes(T, L, a):
        w = V * hid * 2
        kv = NL * 2 * Hkv * L * d * 2
        tree_in = NL * T * (Hq + 2 * Hkv) * d * 2 + T * hid * 2
        tree_kv_out = NL * T * 2 * Hkv * d * 2
        att_out = NL * T * Hq * d * 2
        compact = NL * 2 * (a + 1) * 2 * Hkv * d * 2
        stats = T * 12
        return w + kv + tree_in + tree_kv_out + att_out + compact + stats

    bytes_total = sum(step_bytes(T, L, a) for T, L, a, _, _ in trace)
    lm_bytes = sum(V * hid * 2 + T * hid * 2 for T in lm_T)
    lm_flops = sum(2.0 * T * V * hid for T in lm_T)
    lm_s = sum(lm_ms) / 1e3
    steps_per_s = K / elapsed
    us = elapsed / K * 1e6
    hbm = bytes_total / elapsed / 1e9
    lm_gbps = lm_bytes / lm_s / 1e9
    Tcount = histogram(T for T, *_ in trace)
    accept_mean = float(np.mean([a + 1 for _, _, a, _, _ in trace]))
    switches = sum(1 for i in range(1, len(trace)) if trace[i][4] != trace[i - 1][4])
    log(f"{K} steps in {elapsed:.3f}s: {us:.1f} us/step, {hbm:.0f} GB/s algorithmic; "
        f"LM head {np.mean(lm_ms) * 1e3:.1f} us avg over {len(lm_ms)} launches, {lm_gbps:.0f} GB/s; "
        f"T histogram {Tcount}; mean tokens/step {accept_mean:.3f}; switches {switches}; "
        f"final L {res['L_end']}; LM head us by T {lm_us_by_T}")

    # the other scheduling mode on the same workload, same step count
    other = None
    if args.scheduler == "auto" and on_gpu and not args.graph:
        gc.collect()
        r2 = run.run(K, args.warmup, policy, grow=grows, start_rung=max(args.fixed_topo, 0),
                     arm=not args.no_arm, arm_reach=not fixed, n_events=0, event_pass=0,
                     on_gpu=False)
        other = {"scheduler": "host (one result record read per step, next LM head armed)",
                 "us_per_step": round(r2["elapsed"] / K * 1e6, 2),
                 "steps_per_s": round(K / r2["elapsed"], 2),
                 "hbm_frac": round(sum(step_bytes(T, L, a) for T, L, a, _, _ in r2["trace"])
                                   / r2["elapsed"] / 1e9 / HBM_PEAK_GBPS, 4)}
        log(f"host-scheduled: {other['us_per_step']} us/step")
        # the same device-scheduled steps replayed as captured HIP graph
        # segments (no host launches inside a segment)
        gc.collect()
        r3 = run.run(K, args.warmup, policy, grow=grows, start_rung=max(args.fixed_topo, 0),
                     arm=not args.no_arm, arm_reach=not fixed, n_events=0, event_pass=0,
                     on_gpu=True, graph=True)
        other["graph_replay"] = {"scheduler": "GPU, steps replayed as captured HIP graph segments",
                                 "us_per_step": round(r3["elapsed"] / K * 1e6, 2),
                                 "steps_per_s": round(K / r3["elapsed"], 2)}
        log(f"device-scheduled, graph replay: {other['graph_replay']['us_per_step']} us/step")

    cpu = None
    if not args.no_cpu_baseline and NL == 1:
        cpu = cpu_baseline(args, run, [topo for *_, topo in trace])
    traffic = lm_head_traffic(res["lm_rows"] or [T for T, *_ in trace], on_gpu)
    extras, switching = None, None
    if not args.no_extras:
        extras = next_rows(api, synth, run.W[0], run.pool, hid, V, run.dev)
        if args.workload == "tree27_L256_7b":
            del run
            gc.collect()
            torch.cuda.empty_cache()
            switching = switch_study(args, api, synth, torch)

    line = {
        "metric": METRIC, "value": round(steps_per_s, 2), "unit": "steps/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(elapsed / K * 1e3, 5),
        "us_per_step": round(us, 2), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "hbm_GBps_algorithmic": round(hbm, 1), "hbm_frac": round(hbm / HBM_PEAK_GBPS, 4),
        "config": {"workload": wl.name, "batch": 1, "layers": NL, "heads": Hq, "kv_heads": Hkv,
                   "head_dim": d, "hidden": hid, "vocab": V, "prefix_len_start": wl.prefix_len,
                   "prefix_len_end": res["L_end"] if grows else wl.prefix_len,
                   "prefix": "growing by the accepted tokens" if grows else "reset every step",
                   "bank_T": bank.T,
                   "scheduler": ("hysteretic ladder on=0.8 off=0.6" if not fixed
                                 else f"fixed topo {args.fixed_topo}")
                   + (", on the GPU" if on_gpu else ", on the host"),
                   "T_histogram": {str(k): v for k, v in Tcount.items()},
                   "next_lm_head_armed": bool(not args.no_arm and not on_gpu),
                   "mean_tokens_per_step": round(accept_mean, 4), "topology_switches": switches,
                   "weight_copies": args.weight_copies, "parallelism": "single GPU"},
        "roofline": {"kernel": ("LM head with statistics partials: "
                                + ("lm_head_dyn_small_kernel (tree sized on the GPU) up to 32 nodes, "
                                   "lm_head_dyn_large_kernel above" if on_gpu else
                                   "lm_head_pair_kernel up to 32 nodes, lm_head_hyb_kernel up to 64, "
                                   "lm_head_gemm_kernel above")),
                     "bound": "hbm", "achieved": round(lm_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(lm_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": round(lm_bytes / max(1, len(lm_T))),
                     "avg_us": round(float(np.mean(lm_ms)) * 1e3, 2), "avg_us_by_T": lm_us_by_T,
                     "mfma_TFLOPs": round(lm_flops / lm_s / 1e12, 1),
                     "mfma_frac_bf16": round(lm_flops / lm_s / 1e12 / MFMA_PEAK_BF16_TFLOPS, 4),
                     "timed_launches": len(lm_ms), "timed_launches_in_region": n_in_region,
                     "timing": "HIP events (no system fence) on the step stream around the LM-head "
                               f"launch of a seeded random {n_in_region} of the {K} timed steps and "
                               f"of all {len(lm_ms) - n_in_region} steps of an event pass run right "
                               "after the timed region (same loop, inputs and state); the LM head "
                               "queued behind the previous step's publish kernel or a launch gate, "
                               "so that each pair brackets the kernel"},
        "cpu_baseline": cpu,
        "other_scheduler": other,
        "switching": switching,
        "next_rows": extras,
    }
    print(json.dumps(line), flush=True)


def switch_study(args, api, synth, torch):
    """What switching trees costs: the 5-tree bank at prefix 2048 (reset every
    step), (a) the ladder's own choices, (b) a tree one rung up or down every
    step (a reflecting walk: a switch at every step), and (c) one fixed tree
    per run, every run armed the same way (the next step's LM head sized for
    the next rung).  Overheads are the runs' step times minus the fixed-tree
    step times weighted by the same tree-size histogram."""
    lib = api.lib
    K, W = args.switch_steps, max(10, args.switch_steps // 10)
    run = SingleSeq(api, synth, torch, "bank5_L2048_7b", args.pool, args.weight_copies, 0)
    n, Ts = run.n_topo, run.Ts
    us = lambda r: r["elapsed"] / K * 1e6   # noqa: E731
    lad = run.run(K, W, ladder(lib, n), grow=False)
    g = np.random.default_rng(11)

    def walk(topo, s):
        if topo == 0:
            return 1
        if topo == n - 1:
            return n - 2
        return topo + (1 if g.random() < 0.5 else -1)

    wk = run.run(K, W, walk, grow=False, start_rung=n // 2)
    fixed_us = {}
    for r in range(n):
        fixed_us[Ts[r]] = us(run.run(K, W, lambda topo, s, r=r: r, grow=False, start_rung=r))
    lad2 = run.run(K, W, ladder(lib, n), grow=False)

    def summary(res):
        hist = histogram(T for T, *_ in res["trace"])
        weighted = sum(c * fixed_us[T] for T, c in hist.items()) / K
        sw = sum(1 for i in range(1, K) if res["trace"][i][4] != res["trace"][i - 1][4])
        return hist, weighted, sw

    h_l, w_l, sw_l = summary(lad)
    h_w, w_w, sw_w = summary(wk)
    h_l2, w_l2, _ = summary(lad2)
    lad_over = 0.5 * ((us(lad) - w_l) + (us(lad2) - w_l2))
    out = {"workload": "bank5_L2048_7b", "prefix": "2048, reset every step", "steps_per_run": K,
           "arming": "every run: next LM head sized for the next rung",
           "fixed_tree_us": {str(T): round(v, 2) for T, v in fixed_us.items()},
           "ladder_us": [round(us(lad), 2), round(us(lad2), 2)],
           "ladder_switches": sw_l, "ladder_T_histogram": {str(k): v for k, v in h_l.items()},
           "ladder_fixed_weighted_us": [round(w_l, 2), round(w_l2, 2)],
           "switch_overhead_us": round(lad_over, 2),
           "walk_us": round(us(wk), 2), "walk_switches": sw_w,
           "walk_T_histogram": {str(k): v for k, v in h_w.items()},
           "walk_fixed_weighted_us": round(w_w, 2),
           "walk_overhead_us": round(us(wk) - w_w, 2)}
    log("switching study", json.dumps(out))
    return out


def run_batched(args, api, synth, torch, lib):
    """The batched verification step: 8 sequences, each with its own tree from
    a 5-tree bank (8..128 nodes) and its own prefix (512..16384, growing), GQA
    32:8, vocabulary 128256.  A step, in dependency order on one stream:
    batched tree attention, the LM head with statistics over the
    concatenated rows, batched greedy acceptance and compaction; then the
    host reads every sequence's (accept length, s) in one copy and moves
    every sequence's ladder in one call.  The hidden rows of a step are gathered from a staged pool per
    sequence (the model would hand them over contiguous); the draft tokens
    of every (step, sequence, tree) are drawn before the timed region and a
    step's are written from pinned memory; the attention is issued first, as
    it needs neither."""
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS["batch8_gqa_v128k"]
    B, Hq, Hkv, d, hid, V = 8, wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.hidden, wl.vocab
    trees = synth.workload_trees(wl)
    bank = api.Bank(trees)
    Ts, n_topo, Tmax, Dmax = bank.T, len(trees), max(bank.T), max(bank.D)
    total = args.warmup + args.steps
    lens0 = synth.batch_prefix_lens(wl.ident, B)
    cap = int(lens0.max()) + total * (Dmax + 1) + Tmax + 64
    scale, theta = 1.0 / math.sqrt(d), wl.rope_theta
    bf = torch.bfloat16
    gen = torch.Generator(device=dev)

    def randn(shape, seed, std=1.0):
        gen.manual_seed(seed)
        return (torch.randn(shape, generator=gen, device=dev) * std).to(bf)

    t0 = time.time()
    W = randn((V, hid), 7001, wl.w_std)
    kcs = [torch.zeros((Hkv, cap, d), dtype=bf, device=dev) for _ in range(B)]
    vcs = [torch.zeros((Hkv, cap, d), dtype=bf, device=dev) for _ in range(B)]
    for b in range(B):
        kcs[b][:, : lens0[b]] = randn((Hkv, int(lens0[b]), d), 7100 + 2 * b)
        vcs[b][:, : lens0[b]] = randn((Hkv, int(lens0[b]), d), 7101 + 2 * b)
    # pool: per entry, attention rows for the largest batch, and per sequence
    # slot 128 hidden rows with a confidence regime planted (lift ~ U[11, 18]
    # high or U[0, 11] low, a two-state chain per slot) and their argmax
    P = 8
    rows_max = B * Tmax
    g_np = np.random.default_rng(7)
    hi = g_np.random(B) < 0.5
    pool = []
    lg = torch.empty((Tmax, V), dtype=torch.float32, device=dev)
    amd = torch.empty(Tmax, dtype=torch.int32, device=dev)
    for e in range(P):
        ent = {"q": randn((rows_max, Hq, d), 7200 + 4 * e), "kt": randn((rows_max, Hkv, d), 7201 + 4 * e),
               "vt": randn((rows_max, Hkv, d), 7202 + 4 * e), "x": [], "am": []}
        for b in range(B):
            if g_np.random() >= 0.9:
                hi[b] = not hi[b]
            delta = g_np.uniform(11.0, 18.0) if hi[b] else g_np.uniform(0.0, 11.0)
            x = randn((Tmax, hid), 7300 + 16 * e + b).float()
            spike = torch.from_numpy(g_np.integers(0, V, Tmax)).to(dev)
            x += (delta / (hid * wl.w_std ** 2)) * W.index_select(0, spike).float()
            x = x.to(bf)
            api.verify_logits(x, W, lg)
            api.logit_stats(lg, 1.0, None, None, amd)
            ent["x"].append(x)
            ent["am"].append(amd.cpu().numpy().copy())
        ent["x_all"] = torch.cat(ent["x"])   # [B * Tmax, hid], slot b at rows b * Tmax
        pool.append(ent)
    del lg
    parents = [np.asarray(t, np.int64) for t in trees]
    u_tab = g_np.random((total, rows_max))
    r_tab = g_np.integers(0, V, (total, rows_max)).astype(np.int32)
    # draft tokens of every (step, sequence, tree) and the hidden-row indices
    # of every (sequence, tree), drawn before the timed region (the drafter's
    # output is an input of the step): node i of sequence b takes the
    # target's argmax at its parent with probability p_acc, else a random
    # token (draws from the sequence's slot b * Tmax ..)
    tok_pre = []
    for t in range(total):
        per_b = []
        for b in range(B):
            am_b = pool[t % P]["am"][b]
            u, r = u_tab[t, b * Tmax:(b + 1) * Tmax], r_tab[t, b * Tmax:(b + 1) * Tmax]
            per_k = []
            for k, par in enumerate(parents):
                T = Ts[k]
                tk = np.where(u[:T] < wl.p_acc, am_b[np.maximum(par, 0)], r[:T]).astype(np.int32)
                tk[0] = -1
                per_k.append(tk)
            per_b.append(per_k)
        tok_pre.append(per_b)
    idx_pre = [[b * Tmax + np.arange(Ts[k], dtype=np.int64) for k in range(n_topo)] for b in range(B)]
    log(f"batched workload: B={B}, bank T={Ts}, prefix {lens0.min()}..{lens0.max()}, cap={cap}; "
        f"staged in {time.time() - t0:.1f}s")

    out = torch.empty((rows_max, Hq, d), dtype=bf, device=dev)
    aws = torch.empty(api.tree_attn_batched_workspace(B, Tmax, Hq, Hkv, d, cap), dtype=torch.uint8,
                      device=dev)
    part = torch.empty(lib.entmtp_stats_partials_bytes(rows_max, hid, V), dtype=torch.uint8, device=dev)
    H = torch.empty(rows_max, device=dev)
    p1 = torch.empty(rows_max, device=dev)
    am = torch.empty(rows_max, dtype=torch.int32, device=dev)
    # one pinned staging buffer in (the step's draft tokens, then its hidden-row
    # indices) and one out (accept lengths, then the s the ladder reads): one
    # copy each way per step
    stage_h = torch.empty(2 * rows_max, dtype=torch.int32, pin_memory=True)
    stage_d = torch.empty(2 * rows_max, dtype=torch.int32, device=dev)
    stage_np = stage_h.numpy()
    xg = torch.empty((rows_max, hid), dtype=bf, device=dev)
    cap_path = Dmax + 1
    res_d = torch.zeros(2 * B, dtype=torch.int32, device=dev)
    acc, best = res_d[:B], res_d[B:].view(torch.float32)
    bon = torch.zeros(B, dtype=torch.int32, device=dev)
    path = torch.full((B, cap_path), -1, dtype=torch.int32, device=dev)
    res_h = torch.empty(2 * B, dtype=torch.int32, pin_memory=True)
    res_np = res_h.numpy()
    ev_lm = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    done = torch.cuda.Event()
    # every sequence's tree (its rung on the ladder) and prefix length, int32
    # host arrays handed to the C ABI as they stand
    rung = np.zeros(B, np.int32)
    lens = lens0.astype(np.int32)
    lm_us, trace = [], []
    # The shapes are fixed here, so the binding's tensor checks run once, on
    # the first warmup step (through api.*); every later step calls the C ABI
    # with the same pointers, which a native serving loop would hold.
    P_ = ctypes.c_void_p
    t_p, l_p = rung.ctypes.data_as(P_), lens.ctypes.data_as(P_)
    sv_p = res_np[B:].ctypes.data_as(P_)        # the s of every sequence (float32)
    kp = (P_ * B)(*[k.data_ptr() for k in kcs])
    vp = (P_ * B)(*[v.data_ptr() for v in vcs])
    s_p = P_(torch.cuda.current_stream().cuda_stream)
    ptr = {n: P_(x.data_ptr()) for n, x in (("out", out), ("aws", aws), ("part", part), ("W", W),
                                             ("xg", xg), ("H", H), ("p1", p1), ("am", am),
                                             ("tok", stage_d), ("acc", acc), ("best", best),
                                             ("bon", bon), ("path", path))}
    e_ptr = [{n: P_(ent[n].data_ptr()) for n in ("q", "kt", "vt")} for ent in pool]
    aws_bytes, part_bytes = aws.numel(), part.numel()
    idx_cache = {}

    def call(rc):
        if rc:
            raise RuntimeError(api.last_error())

    def step(t, timed_lm, checked=False):
        e, ep = pool[t % P], e_ptr[t % P]
        topo = [int(k) for k in rung]
        R = sum(Ts[k] for k in topo)
        if checked:
            api.tree_attn_batched(bank, topo, lens.tolist(), e["q"][:R], e["kt"][:R], e["vt"][:R],
                                  kcs, vcs, scale, theta, out[:R], aws)
        else:
            call(lib.entmtp_tree_attn_batched(bank.handle, B, t_p, l_p, ep["q"], ep["kt"], ep["vt"],
                                              kp, vp, cap, Hq, Hkv, d, scale, theta, ptr["out"],
                                              ptr["aws"], aws_bytes, s_p))
        # draft tokens and the hidden-row gather for this batch layout, staged
        # while the attention runs
        key = tuple(topo)
        idx = idx_cache.get(key)
        if idx is None:
            idx = idx_cache[key] = np.concatenate([idx_pre[b][k] for b, k in enumerate(topo)])
        stage_np[:R] = np.concatenate([tok_pre[t][b][k] for b, k in enumerate(topo)])
        stage_np[rows_max:rows_max + R] = idx
        stage_d.copy_(stage_h, non_blocking=True)
        torch.index_select(e["x_all"], 0, stage_d[rows_max:rows_max + R], out=xg[:R])
        if timed_lm:
            ev_lm[0].record()
        call(lib.entmtp_verify_logits_partials(ptr["xg"], ptr["W"], R, hid, V, 1.0, None, ptr["part"],
                                               part_bytes, s_p))
        if timed_lm:
            ev_lm[1].record()
        if checked:
            api.stats_finalize(part, R, V, 1.0, H, p1, am)
            api.accept_batched(bank, topo, stage_d[:R], am, p1, acc, path, bon, best)
            api.kv_compact_batched(path, acc, lens.tolist(), kcs, vcs)
        else:
            call(lib.entmtp_stats_finalize(ptr["part"], R, V, 1.0, ptr["H"], ptr["p1"], ptr["am"], s_p))
            call(lib.entmtp_accept_batched(bank.handle, B, t_p, ptr["tok"], ptr["am"], ptr["p1"],
                                           ptr["acc"], ptr["path"], cap_path, ptr["bon"], ptr["best"],
                                           s_p))
            call(lib.entmtp_kv_compact_batched(B, ptr["path"], cap_path, ptr["acc"], l_p, kp, vp, 1,
                                               Hkv * cap * d, Hkv, cap, d, s_p))
        res_h.copy_(res_d, non_blocking=True)
        done.record()
        done.synchronize()
        a = res_np[:B]
        if timed_lm:
            lm_us.append((R, ev_lm[0].elapsed_time(ev_lm[1]) * 1e3))
        trace.append((R, int(a.sum()) + B))
        np.add(lens, a + 1, out=lens)
        call(lib.entmtp_ladder_next_batched(B, t_p, sv_p, n_topo, 0.8, 0.6))

    for t in range(args.warmup):
        step(t, False, checked=t == 0)
    trace.clear()
    torch.cuda.synchronize()
    gc.disable()
    t_start = time.perf_counter()
    for t in range(args.warmup, total):
        step(t, (t - args.warmup) % args.event_every == 0)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    gc.enable()
    K = args.steps
    us = elapsed / K * 1e6
    tokens = sum(n for _, n in trace)
    rows_mean = float(np.mean([R for R, _ in trace]))
    lm_mean = float(np.mean([u for _, u in lm_us]))
    lm_rows = float(np.mean([R for R, _ in lm_us]))
    lm_bytes = V * hid * 2
    lm_flops = 2.0 * lm_rows * V * hid
    log(f"{K} batched steps in {elapsed:.3f}s: {us:.1f} us/step, {tokens / elapsed:.0f} tokens/s, "
        f"mean rows {rows_mean:.1f}, LM head {lm_mean:.1f} us at {lm_rows:.0f} rows")
    line = {
        "metric": METRIC, "value": round(K / elapsed, 2), "unit": "steps/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(elapsed / K * 1e3, 5), "us_per_step": round(us, 2),
        "tokens_per_s": round(tokens / elapsed, 1), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "heads": Hq, "kv_heads": Hkv, "head_dim": d,
                   "hidden": hid, "vocab": V, "prefix_len_start": [int(x) for x in lens0],
                   "bank_T": Ts, "mean_rows_per_step": round(rows_mean, 1),
                   "mean_tokens_per_step": round(tokens / K, 3),
                   "scheduler": "hysteretic ladder on=0.8 off=0.6 per sequence, on the host",
                   "parallelism": "single GPU"},
        "roofline": {"kernel": "LM head with statistics partials over the batch's rows",
                     "bound": "hbm", "achieved": round(lm_bytes / lm_mean / 1e3, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(lm_bytes / lm_mean / 1e3 / HBM_PEAK_GBPS, 4), "traffic": None,
                     "avg_us": round(lm_mean, 2), "mean_rows": round(lm_rows, 1),
                     "mfma_TFLOPs": round(lm_flops / lm_mean / 1e6, 1),
                     "mfma_frac_bf16": round(lm_flops / lm_mean / 1e6 / MFMA_PEAK_BF16_TFLOPS, 4),
                     "timing": "HIP events around the LM-head launch of every n-th timed step"},
        "cpu_baseline": None,
    }
    print(json.dumps(line))


def next_rows(api, synth, W, pool, hid, V, dev, reps=50):
    """Timings (HIP events, after the timed region) of the kernels beyond the
    greedy step: typical and speculative-sampling acceptance on a 26-node tree
    at these shapes, and the frontier scoring of the offline search at its
    rollout size (100 prompts x 256 tokens of samples over a 64-node tree and
    its frontier)."""
    import torch
    out = {}
    # typical acceptance (T 0.7, eps 0.09, alpha 0.3): draft logits + the walk
    tree = synth.uniform_attach_tree(3, 26, 4)
    bank = api.Bank([tree])
    T = len(tree)
    X = pool[0]["x"][:T]
    lg = torch.empty((T, V), dtype=torch.float32, device=dev)
    H, p1 = torch.empty(T, device=dev), torch.empty(T, device=dev)
    am = torch.empty(T, dtype=torch.int32, device=dev)
    ws = torch.empty(api.verify_logits_stats_workspace(T, hid, V), dtype=torch.uint8, device=dev)
    api.verify_logits_stats(X, W, lg, 1 / 0.7, H, p1, am, ws)
    tok = am[torch.tensor([max(p, 0) for p in tree], device=dev)].contiguous()
    zd, zt = torch.empty(T, device=dev), torch.empty(T, device=dev)
    a = torch.zeros(1, dtype=torch.int32, device=dev)
    path = torch.zeros(32, dtype=torch.int32, device=dev)
    bonus = torch.zeros(1, dtype=torch.int32, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    out["typical_draft_logits_us"] = round(timed(
        lambda: api.draft_logits(bank, 0, X, W, tok, am, zd, zt)), 2)
    out["typical_accept_us"] = round(timed(
        lambda: api.accept_typical(bank, 0, tok, am, zd, zt, H, p1, 1 / 0.7, 0.09, 0.3, a, path,
                                   bonus)), 2)
    out["typical_tree_nodes"] = T
    # speculative sampling on the same tree: logits, a draft distribution per
    # node (softmax of perturbed logits) and uniforms
    gq = torch.Generator(device="cpu").manual_seed(5)
    qd = torch.softmax(lg + torch.randn(lg.shape, generator=gq).to(dev), dim=1).contiguous()
    ua = torch.rand(T, generator=gq).to(dev)
    usd = torch.rand(T, generator=gq).to(dev)
    wsp = torch.empty(V, dtype=torch.float32, device=dev)
    out["stochastic_accept_us"] = round(timed(
        lambda: api.accept_stochastic(bank, 0, tok, lg, qd, 1 / 0.7, am, p1, ua, usd, wsp, a,
                                      path, bonus)), 2)
    # frontier scoring at rollout size
    parent = synth.uniform_attach_tree(79, 64, 5)
    joint, in_tree = api.frontier_tree(parent, 6)
    fb = api.Bank([joint])
    J, S = len(joint), 100 * 256
    g = torch.Generator(device="cpu").manual_seed(7)
    ok = (torch.rand((S, J), generator=g) < 0.7).to(torch.uint8).to(dev)
    it = torch.tensor(in_tree, dtype=torch.uint8, device=dev)
    sums = torch.zeros(J, dtype=torch.int32, device=dev)
    best = torch.zeros(1, dtype=torch.int32, device=dev)
    us = timed(lambda: api.frontier_score(fb, 0, it, sums, best, local_ok=ok))
    out["frontier_score_us"] = round(us, 2)
    out["frontier_samples"] = S
    out["frontier_joint_nodes"] = J
    out["frontier_samples_per_s"] = round(S / (us * 1e-6), 1)
    return out


def lm_head_traffic(Ts, on_gpu=False):
    """Measured HBM bytes per LM-head launch (FETCH_SIZE + WRITE_SIZE, scaled by
    a device-copy calibration) for this step mix, from the committed counter
    record -- or None when the kernel sources changed since it was taken or
    the record lacks a kernel the mix launches."""
    from paper_2606_27550_amd import rocprof_summary
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "lm_head_traffic.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("lm_head_source_sha256") != rocprof_summary.lm_head_source_hash():
        return None
    per = {}
    for name, v in rec["per_variant"].items():
        targs = [x.strip() for x in name.split("<")[1].rstrip(">").split(",")]
        kernel = name.split("<")[0].split()[-1]
        if kernel == "lm_head_pair_kernel":            # <NT, NCH>: up to 32 nodes
            key = (kernel, int(targs[0]))
        elif kernel == "lm_head_hyb_kernel" and targs[3] == "true":   # <NT, S, NCH, STATS, WT>
            key = (kernel, int(targs[0]))
            # large tiles: the step pairs slices per workgroup (last argument
            # 2); an unpaired launch of the entry points must not stand in
            if key in per and len(targs) > 4 and targs[4] != "2":
                continue
        elif kernel == "lm_head_gemm_kernel" and targs[-1] == "true":   # <BM, BN, NW, NST, STATS>
            key = (kernel, 0)
        elif kernel in ("lm_head_dyn_small_kernel", "lm_head_dyn_large_kernel"):
            key = (kernel, 0)
        else:
            continue
        per[key] = v["fetch_bytes"] + v["write_bytes"]
    tot = 0.0
    for T in Ts:
        if on_gpu:   # the device-sized kernels: the small one up to 32 nodes
            key = ("lm_head_dyn_small_kernel" if T <= 32 else "lm_head_dyn_large_kernel", 0)
        elif T <= 32:
            key = ("lm_head_pair_kernel", 1 if T <= 16 else 2)
        elif T <= 64:
            key = ("lm_head_hyb_kernel", 4)
        else:   # the tiled kernel where it takes the launch, else the 128-node streaming tile
            key = ("lm_head_gemm_kernel", 0) if ("lm_head_gemm_kernel", 0) in per else ("lm_head_hyb_kernel", 8)
        if key not in per:
            return None
        tot += per[key]
    return round(tot / len(Ts))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(args, run, topo_seq):
    """The oracle, as it stands, on a bounded sample of the same workload: the
    timed run's own sequence of trees, from its start, at the starting prefix,
    until the time budget (at least three steps; the median step time is
    reported), then the first tree of that sequence on one host thread."""
    from oracle import entmtp_oracle as orc
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threadpool_limits = None
        threads = os.cpu_count() or 1
    wl, trees, pool = run.wl, run.trees, run.pool
    Hkv, d, L0 = wl.n_kv_heads, wl.head_dim, wl.prefix_len
    order = list(topo_seq) or list(range(len(trees)))
    kc = np.zeros((Hkv, L0 + 256, d), np.uint16)
    vc = np.zeros_like(kc)
    kc[:, :L0], vc[:, :L0] = run.kc0_host, run.vc0_host

    def one(i, k):
        e = pool[i % len(pool)]
        q, kt, vt, x = e["host"]
        T = len(trees[k])
        t0 = time.perf_counter()
        orc.verify_step(trees[k], q[:T], kt[:T], vt[:T], kc, vc, L0, x[:T], run.w_host,
                        e["tok"][k], run.scale, run.theta)
        return time.perf_counter() - t0

    times, done = [], []
    for i, k in enumerate(order):
        times.append(one(i, k))
        done.append(len(trees[k]))
        if sum(times) > args.cpu_budget_s and len(times) >= 3:
            break
    one_thread = []
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            while len(one_thread) < 3 and sum(one_thread) < args.cpu_budget_s / 2:
                one_thread.append(one(0, order[0]))
    hist = histogram(done)
    med = float(np.median(times))
    return {"value": round(1.0 / med, 4), "unit": "steps/s", "cores": threads, "kind": "oracle",
            "affinity_cores": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
            "median_step_s": round(med, 4),
            "value_1thread": round(1.0 / float(np.median(one_thread)), 4) if one_thread else None,
            "steps_1thread": len(one_thread),
            "sample": f"the first {len(done)} steps of the timed run's tree sequence of {wl.name} "
                      f"(tree-size histogram {hist}) at prefix {L0}, {sum(times):.1f}s, value = 1 / "
                      f"median step time; fp64 numpy/BLAS on {threads} host threads; value_1thread: "
                      f"{len(one_thread)} steps of tree {order[0]} on one thread"}


if __name__ == "__main__":
    main()
