// One verification step, end to end, behind a small native context.
//
// The decode loop of §4 verifies the scheduled tree, accepts the longest
// matching path, updates the cache, and reads one scalar back to the host to
// pick the next tree ("Cost": a single device-to-host read per step).  The
// context below validates the fixed sizes once; each step is then a short
// burst of launches.
//
// Host-scheduled steps run as two chains.  The caller's stream carries what
// the next tree choice waits for: the LM head and the statistics merge with
// acceptance, which publishes its result (accept length, bonus token, s and
// the accepted path) into coherent pinned host memory that the host polls
// instead of synchronising a stream.  A side stream carries the cache work:
// the attention layers of the step, preceded by the compaction of the step
// before it.  The head reads the tree's final hidden states, not the cache,
// so nothing on the caller's stream waits for the side stream; the only
// order the cache needs -- step t's compaction before step t+1's attention --
// is the side stream's own, and the compaction takes the accepted path from
// the host record in its launch arguments.  So the next LM head starts as
// soon as the host has chosen the tree, while the previous step's compaction
// and the next attention run beside it.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <vector>

#include "common.hpp"
#include "stats.hpp"

using namespace entmtp;

struct entmtp_step {
  const entmtp_bank* bank = nullptr;
  entmtp_step_config cfg{};
  int32_t T_max = 0;
  int32_t D_max = 0;
  size_t attn_bytes = 0;       // attention workspace, at the start of cfg.workspace
  size_t part_offset = 0;      // LM-head statistics partials follow it
  size_t part_bytes = 0;
  size_t dev_offset = 0;       // then the device-scheduled state: DevStep[kRing], DevTopo[K],
  size_t ring_offset = 0;      // and the acceptance ring: kRing x (accept_len, path[path_capacity])
  DevAttnShape dshape;         // attention grids for a tree chosen on the device
  // device-scheduled steps: step t reads state slot t % kRing and writes slot
  // (t + 1) % kRing; its accept length and path go to ring slot t % kRing.
  // Before step t's acceptance writes those slots, the side stream must be
  // done with their previous users (its work of step t + 2 - kRing); the
  // caller's stream waits for the side stream's step t - kWaitLag at every
  // kWaitEvery-th step, which covers the kWaitEvery steps from there
  // (t + kWaitEvery - 1 + 2 - kRing <= t - kWaitLag) with one wait packet.
  static constexpr int kRing = 16;
  static constexpr int kWaitEvery = 8;
  static constexpr int kWaitLag = 4;
  static_assert(kWaitEvery + 1 - kRing <= -kWaitLag, "ring too shallow for the wait cadence");
  bool dev_started = false;
  uint64_t dev_t = 0;          // steps launched since entmtp_step_device_start
  uint64_t dev_compact = 0;    // steps whose compaction has been enqueued
  uint64_t dev_sync_t = 0;     // steps whose side-stream work the caller's stream has joined
  hipEvent_t ev_side[kRing] = {};   // side-stream work of device-scheduled step t done
  StepMirror* host = nullptr;  // pinned, coherent
  StepMirror* dev = nullptr;   // device address of `host`
  // launch gate for timed LM heads: a pinned, coherent word the host writes
  // once the LM head is enqueued (its own 64-byte line)
  uint32_t* gate_host = nullptr;
  uint32_t* gate_dev = nullptr;
  uint32_t gate_seq = 0;
  // the next step's LM head, enqueued ahead of its launch behind the gate
  // (entmtp_step_arm): the rows it covers and the inputs it reads
  bool armed = false;
  int32_t armed_T = 0;
  int32_t armed_parts = 0;     // statistics partials per node it writes
  int32_t lm_parts = 0;        // the same for the LM head of the latest launch
  const void* armed_hidden = nullptr;
  const void* armed_w = nullptr;
  hipStream_t side = nullptr;  // attention chain (default priority, non-blocking)
  hipEvent_t fork = nullptr;   // caller's stream -> side stream
  hipEvent_t join = nullptr;   // side stream -> caller's stream
  uint32_t seq = 0;            // sequence number of the latest launch
  bool pending = false;        // a launched step whose result has not been read
  int32_t pending_L = 0;       // its prefix length
  // the compaction of the latest step whose result was read, not yet enqueued
  bool compact_due = false;
  int32_t due_L = 0, due_a = 0;
  int32_t due_path[ENTMTP_D_MAX + 1] = {};
};

namespace {

size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

// The longest a launch gate holds its stream: 2 ms of the 100 MHz constant
// clock (wall_clock64).
constexpr uint64_t kGateTicks = 200000;

// Holds the stream until the host has stored `want` to the pinned word, which
// it does right after enqueuing the work behind the gate, or until max_ticks
// have passed.  A timing event recorded behind the gate is therefore stamped
// with the timed kernel already in the queue; recorded on an idle stream, it
// would be stamped before the host's launch call and count that call's time
// and the idle queue's dispatch latency as the kernel's.
__global__ void launch_gate_kernel(const uint32_t* word, uint32_t want, uint64_t max_ticks) {
  if (threadIdx.x != 0) return;
  const uint64_t t0 = wall_clock64();
  while (__hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != want &&
         wall_clock64() - t0 < max_ticks)
    __builtin_amdgcn_s_sleep(2);
}

// Lets the gated work of the latest gate kernel run (harmless if it already
// has, or if the gate's time limit ended the wait).
void open_gate(entmtp_step* st) {
  __atomic_store_n(st->gate_host, st->gate_seq, __ATOMIC_RELEASE);
}

// Enqueues a gate kernel on s with a fresh sequence number.
int32_t enqueue_gate(entmtp_step* st, hipStream_t s) {
  st->gate_seq = st->gate_seq + 1u == 0u ? 1u : st->gate_seq + 1u;
  hipLaunchKernelGGL(launch_gate_kernel, dim3(1), dim3(64), 0, s, st->gate_dev, st->gate_seq,
                     kGateTicks);
  return launch_status("launch gate");
}

void bank_extent(const entmtp_bank* bank, int32_t* T_max, int32_t* D_max) {
  int32_t t = 0, dd = 0;
  for (const TopoDesc& d : bank->desc) {
    t = d.T > t ? d.T : t;
    dd = d.D > dd ? d.D : dd;
  }
  *T_max = t;
  *D_max = dd;
}

// Workspace split for a validated configuration; returns the total bytes.
size_t layout(const entmtp_step_config& c, int32_t T_max, int32_t n_topo, size_t* attn,
              size_t* part_off, size_t* part, size_t* dev_off, size_t* ring_off) {
  *attn = entmtp_tree_attn_workspace(T_max, c.Hq, c.Hkv, c.d, c.cap);
  *part_off = round256(*attn);
  *part = entmtp_stats_partials_bytes(T_max, c.hid, c.V);
  *dev_off = round256(*part_off + *part);
  *ring_off = *dev_off + round256(entmtp_step::kRing * sizeof(DevStep) +
                                  static_cast<size_t>(n_topo) * sizeof(DevTopo));
  return *ring_off + round256(static_cast<size_t>(entmtp_step::kRing) *
                              (1 + std::max(c.path_capacity, 1)) * sizeof(int32_t));
}

bool finite_positive(float x) { return x > 0.f && std::isfinite(x); }

// Validates everything but the workspace pointer (its size is what the
// workspace query answers).
int32_t check_config(const entmtp_bank* bank, const entmtp_step_config* c, int32_t* T_max,
                     int32_t* D_max) {
  if (int32_t rc = check_device_bank(bank, 0)) return rc;
  ENTMTP_CHECK_ARG(c != nullptr, ENTMTP_EINVAL, "config is NULL");
  bank_extent(bank, T_max, D_max);
  ENTMTP_CHECK_ARG(c->n_layers >= 1, ENTMTP_EINVAL, "n_layers = %d < 1", c->n_layers);
  ENTMTP_CHECK_ARG(c->d == ENTMTP_HEAD_DIM, ENTMTP_EINVAL, "head dim %d unsupported (built for %d)",
                   c->d, ENTMTP_HEAD_DIM);
  ENTMTP_CHECK_ARG(c->Hq >= 1 && c->Hkv >= 1, ENTMTP_EINVAL, "Hq = %d, Hkv = %d must be >= 1",
                   c->Hq, c->Hkv);
  ENTMTP_CHECK_ARG(c->Hq % c->Hkv == 0, ENTMTP_ERANGE, "Hq = %d is not a multiple of Hkv = %d",
                   c->Hq, c->Hkv);
  ENTMTP_CHECK_ARG(c->tree_rows >= *T_max, ENTMTP_EINVAL,
                   "tree_rows = %d below the bank's largest tree (%d nodes)", c->tree_rows, *T_max);
  ENTMTP_CHECK_ARG(c->cap >= *T_max, ENTMTP_ERANGE, "cap = %d below the largest tree (%d nodes)",
                   c->cap, *T_max);
  ENTMTP_CHECK_ARG(finite_positive(c->scale), ENTMTP_EINVAL, "scale must be positive and finite");
  ENTMTP_CHECK_ARG(c->rope_theta >= 0.f && std::isfinite(c->rope_theta), ENTMTP_EINVAL,
                   "rope_theta must be >= 0 and finite");
  ENTMTP_CHECK_ARG(c->k_cache && c->v_cache && aligned16(c->k_cache) && aligned16(c->v_cache),
                   ENTMTP_EINVAL, "caches must be non-NULL and 16-byte aligned");
  ENTMTP_CHECK_ARG(c->n_layers == 1 ||
                       (c->cache_layer_stride >= static_cast<int64_t>(c->Hkv) * c->cap * c->d &&
                        c->cache_layer_stride % 8 == 0),
                   ENTMTP_EINVAL, "cache_layer_stride %lld must cover one layer and keep alignment",
                   static_cast<long long>(c->cache_layer_stride));
  ENTMTP_CHECK_ARG(c->w_lm && aligned16(c->w_lm), ENTMTP_EINVAL, "w_lm must be non-NULL and aligned");
  ENTMTP_CHECK_ARG(c->V >= 1, ENTMTP_EINVAL, "V = %d < 1", c->V);
  ENTMTP_CHECK_ARG(entmtp_stats_partials_bytes(*T_max, c->hid, c->V) > 0, ENTMTP_EINVAL,
                   "hid = %d: the step needs a multiple of 512", c->hid);
  ENTMTP_CHECK_ARG(finite_positive(c->inv_temp), ENTMTP_EINVAL, "inv_temp must be positive and finite");
  ENTMTP_CHECK_ARG(aligned16(c->logits) && c->entropy && c->top1p && c->argmax, ENTMTP_EINVAL,
                   "statistics outputs must be non-NULL and logits (if any) 16-byte aligned");
  ENTMTP_CHECK_ARG(c->accept_len && c->bonus && c->best_top1p && c->path, ENTMTP_EINVAL,
                   "acceptance outputs must be non-NULL");
  ENTMTP_CHECK_ARG(c->path_capacity >= *D_max + 1 && c->path_capacity <= ENTMTP_D_MAX + 1,
                   ENTMTP_EINVAL, "path_capacity = %d outside [1 + the bank's depth %d, %d]",
                   c->path_capacity, *D_max, ENTMTP_D_MAX + 1);
  ENTMTP_CHECK_ARG(c->device_prefix_fixed == 0 || c->device_prefix_fixed == 1, ENTMTP_EINVAL,
                   "device_prefix_fixed = %d must be 0 or 1", c->device_prefix_fixed);
  ENTMTP_CHECK_ARG(c->tau_off <= c->tau_on, ENTMTP_EINVAL, "tau_off %g > tau_on %g",
                   static_cast<double>(c->tau_off), static_cast<double>(c->tau_on));
  return ENTMTP_OK;
}

}  // namespace

extern "C" size_t entmtp_step_workspace(const entmtp_bank* bank, const entmtp_step_config* cfg) {
  int32_t T_max = 0, D_max = 0;
  if (check_config(bank, cfg, &T_max, &D_max) != ENTMTP_OK) {
    clear_error();
    return 0;
  }
  size_t attn = 0, off = 0, part = 0, doff = 0, roff = 0;
  const size_t total = layout(*cfg, T_max, static_cast<int32_t>(bank->desc.size()), &attn, &off,
                              &part, &doff, &roff);
  return attn && part ? total : 0;
}

extern "C" int32_t entmtp_step_create(const entmtp_bank* bank, const entmtp_step_config* cfg,
                                      entmtp_step** out) {
  clear_error();
  ENTMTP_CHECK_ARG(out != nullptr, ENTMTP_EINVAL, "out is NULL");
  *out = nullptr;
  int32_t T_max = 0, D_max = 0;
  if (int32_t rc = check_config(bank, cfg, &T_max, &D_max)) return rc;
  size_t attn = 0, off = 0, part = 0, doff = 0, roff = 0;
  const size_t total = layout(*cfg, T_max, static_cast<int32_t>(bank->desc.size()), &attn, &off,
                              &part, &doff, &roff);
  ENTMTP_CHECK_ARG(attn > 0 && part > 0, ENTMTP_EINVAL, "unsupported attention or LM-head sizes");
  ENTMTP_CHECK_ARG(cfg->workspace && (reinterpret_cast<uintptr_t>(cfg->workspace) & 255u) == 0,
                   ENTMTP_EINVAL, "workspace must be non-NULL and 256-byte aligned");
  ENTMTP_CHECK_ARG(cfg->workspace_bytes >= total, ENTMTP_ENOSPC,
                   "workspace has %zu bytes, needs %zu", cfg->workspace_bytes, total);
  int dev = -1;
  if (int32_t rc = hip_status(hipGetDevice(&dev), "hipGetDevice")) return rc;
  ENTMTP_CHECK_ARG(dev == bank->device, ENTMTP_EINVAL,
                   "current device %d differs from the bank's device %d", dev, bank->device);

  entmtp_step* st = new entmtp_step;
  st->bank = bank;
  st->cfg = *cfg;
  st->T_max = T_max;
  st->D_max = D_max;
  st->attn_bytes = attn;
  st->part_offset = off;
  st->part_bytes = part;
  st->dev_offset = doff;
  st->ring_offset = roff;
  void* h = nullptr;
  int32_t rc = hip_status(hipHostMalloc(&h, sizeof(StepMirror), hipHostMallocMapped | hipHostMallocCoherent),
                          "hipHostMalloc (step result record)");
  if (rc == ENTMTP_OK) {
    st->host = static_cast<StepMirror*>(h);
    std::memset(st->host, 0, sizeof(StepMirror));
    void* d = nullptr;
    rc = hip_status(hipHostGetDevicePointer(&d, h, 0), "hipHostGetDevicePointer");
    st->dev = static_cast<StepMirror*>(d);
  }
  if (rc == ENTMTP_OK) {
    void* g = nullptr;
    rc = hip_status(hipHostMalloc(&g, 64, hipHostMallocMapped | hipHostMallocCoherent),
                    "hipHostMalloc (launch gate)");
    if (rc == ENTMTP_OK) {
      st->gate_host = static_cast<uint32_t*>(g);
      *st->gate_host = 0u;
      void* d = nullptr;
      rc = hip_status(hipHostGetDevicePointer(&d, g, 0), "hipHostGetDevicePointer");
      st->gate_dev = static_cast<uint32_t*>(d);
    }
  }
  if (rc == ENTMTP_OK)
    rc = hip_status(hipStreamCreateWithFlags(&st->side, hipStreamNonBlocking), "hipStreamCreate");
  if (rc == ENTMTP_OK)
    rc = hip_status(hipEventCreateWithFlags(&st->fork, hipEventDisableTiming), "hipEventCreate");
  if (rc == ENTMTP_OK)
    rc = hip_status(hipEventCreateWithFlags(&st->join, hipEventDisableTiming), "hipEventCreate");
  for (int k = 0; k < entmtp_step::kRing && rc == ENTMTP_OK; ++k)
    rc = hip_status(hipEventCreateWithFlags(&st->ev_side[k], hipEventDisableTiming),
                    "hipEventCreate");
  if (rc == ENTMTP_OK) {  // the bank's descriptors for device-scheduled steps
    std::vector<DevTopo> topos(bank->desc.size());
    for (size_t k = 0; k < topos.size(); ++k) {
      const TopoDesc& d = bank->desc[k];
      topos[k] = DevTopo{};
      topos[k].T = d.T;
      topos[k].D = d.D;
      topos[k].off_parent = static_cast<int>(d.off_parent);
      topos[k].off_depth = static_cast<int>(d.off_depth);
      topos[k].off_mask = static_cast<int>(d.off_mask);
      topos[k].off_path = static_cast<int>(d.off_path);
    }
    attn_device_splits(bank, cfg->Hq, cfg->Hkv, topos.data());
    auto* dst = static_cast<uint8_t*>(cfg->workspace) + doff + entmtp_step::kRing * sizeof(DevStep);
    rc = hip_status(hipMemcpyAsync(dst, topos.data(), topos.size() * sizeof(DevTopo),
                                   hipMemcpyHostToDevice, static_cast<hipStream_t>(cfg->stream)),
                    "hipMemcpyAsync (bank descriptors)");
    if (rc == ENTMTP_OK)
      rc = hip_status(hipStreamSynchronize(static_cast<hipStream_t>(cfg->stream)),
                      "hipStreamSynchronize");
  }
  if (rc == ENTMTP_OK) rc = attn_device_shape(bank, cfg->Hq, cfg->Hkv, cfg->cap, &st->dshape);
  if (rc != ENTMTP_OK) {
    entmtp_step_destroy(st);
    return rc;
  }
  *out = st;
  return ENTMTP_OK;
}

extern "C" void entmtp_step_destroy(entmtp_step* st) {
  if (!st) return;
  if (st->armed && st->gate_host) {   // the gate kernel must be done with the word before it is freed
    open_gate(st);
    (void)hipStreamSynchronize(static_cast<hipStream_t>(st->cfg.stream));
  }
  if (st->side) (void)hipStreamSynchronize(st->side);
  for (int k = 0; k < entmtp_step::kRing; ++k)
    if (st->ev_side[k]) (void)hipEventDestroy(st->ev_side[k]);
  if (st->join) (void)hipEventDestroy(st->join);
  if (st->fork) (void)hipEventDestroy(st->fork);
  if (st->side) (void)hipStreamDestroy(st->side);
  if (st->host) (void)hipHostFree(st->host);
  if (st->gate_host) (void)hipHostFree(st->gate_host);
  delete st;
}

namespace {

// Enqueues the compaction the host holds (if any) on the side stream.
int32_t enqueue_due_compaction(entmtp_step* st) {
  if (!st->compact_due) return ENTMTP_OK;
  const entmtp_step_config& c = st->cfg;
  st->compact_due = false;
  return launch_compact_host(st->due_path, st->due_a, st->due_L, c.k_cache, c.v_cache, c.n_layers,
                             c.cache_layer_stride, c.Hkv, c.cap, c.d, st->side);
}

DevStep* dev_state(entmtp_step* st) {
  return reinterpret_cast<DevStep*>(static_cast<uint8_t*>(st->cfg.workspace) + st->dev_offset);
}

int32_t* dev_ring(entmtp_step* st, uint64_t t) {
  return reinterpret_cast<int32_t*>(static_cast<uint8_t*>(st->cfg.workspace) + st->ring_offset) +
         (t % entmtp_step::kRing) * (1 + static_cast<size_t>(st->cfg.path_capacity));
}

// Device-scheduled step t's compaction, on the side stream (already ordered
// after its acceptance).
int32_t enqueue_device_compaction(entmtp_step* st, uint64_t t) {
  const entmtp_step_config& c = st->cfg;
  int32_t* ring = dev_ring(st, t);
  st->dev_compact = t + 1;
  return launch_compact_device(dev_state(st) + t % entmtp_step::kRing, ring + 1, c.path_capacity,
                               ring, c.k_cache, c.v_cache, c.n_layers, c.cache_layer_stride, c.Hkv,
                               c.cap, c.d, st->side);
}

int32_t flush_side(entmtp_step* st) {
  ENTMTP_CHECK_ARG(!st->pending, ENTMTP_EINVAL,
                   "a launched step's result has not been read (entmtp_step_wait)");
  if (st->armed) open_gate(st);   // an armed LM head may run now (it stays armed)
  if (int32_t rc = enqueue_due_compaction(st)) return rc;
  if (st->dev_started && st->dev_compact < st->dev_t) {   // the last device-scheduled step's
    auto s = static_cast<hipStream_t>(st->cfg.stream);
    if (int32_t rc = hip_status(hipEventRecord(st->fork, s), "hipEventRecord (fork)")) return rc;
    if (int32_t rc = hip_status(hipStreamWaitEvent(st->side, st->fork, 0), "hipStreamWaitEvent"))
      return rc;
    if (int32_t rc = enqueue_device_compaction(st, st->dev_t - 1)) return rc;
  }
  st->dev_sync_t = st->dev_t;
  if (int32_t rc = hip_status(hipEventRecord(st->join, st->side), "hipEventRecord (join)")) return rc;
  return hip_status(hipStreamWaitEvent(static_cast<hipStream_t>(st->cfg.stream), st->join, 0),
                    "hipStreamWaitEvent");
}

}  // namespace

extern "C" int32_t entmtp_step_flush(entmtp_step* st) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr, ENTMTP_EINVAL, "step is NULL");
  return flush_side(st);
}

extern "C" int32_t entmtp_step_launch(entmtp_step* st, int32_t topo, int32_t prefix_len,
                                      const entmtp_bf16* q, const entmtp_bf16* k_tree,
                                      const entmtp_bf16* v_tree, entmtp_bf16* out,
                                      const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                      const int32_t* draft_tokens, void* ev_lm_begin,
                                      void* ev_lm_end) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr, ENTMTP_EINVAL, "step is NULL");
  ENTMTP_CHECK_ARG(!st->pending, ENTMTP_EINVAL,
                   "the previous step's result has not been read (entmtp_step_wait)");
  const entmtp_step_config& c = st->cfg;
  if (int32_t rc = check_device_bank(st->bank, topo)) return rc;
  if (st->dev_started) {   // device-scheduled steps before this one finish their cache work
    if (int32_t rc = flush_side(st)) return rc;
    st->dev_started = false;
  }
  ENTMTP_CHECK_ARG(q && k_tree && v_tree && out && hidden && draft_tokens, ENTMTP_EINVAL,
                   "per-step inputs and outputs must be non-NULL");
  const int32_t T = st->bank->desc[topo].T;
  ENTMTP_CHECK_ARG(prefix_len >= 0 && static_cast<int64_t>(prefix_len) + T <= c.cap, ENTMTP_ERANGE,
                   "prefix_len %d + T %d outside the cache capacity %d", prefix_len, T, c.cap);
  ENTMTP_CHECK_ARG(w_lm == nullptr || aligned16(w_lm), ENTMTP_EINVAL, "w_lm must be 16-byte aligned");
  auto s = static_cast<hipStream_t>(c.stream);
  uint8_t* ws = static_cast<uint8_t*>(c.workspace);
  void* part = ws + st->part_offset;

  const void* w_step = w_lm ? w_lm : c.w_lm;
  // an armed step: the LM head waits in the stream behind the gate (with the
  // fork recorded ahead of it); opening the gate is the whole launch, unless
  // the tree outgrew the rows it was armed for or its inputs differ (then a
  // fresh LM head follows it and overwrites its partials)
  bool lm_ready = false;
  if (st->armed) {
    ENTMTP_CHECK_ARG(ev_lm_begin == nullptr && ev_lm_end == nullptr, ENTMTP_EINVAL,
                     "the LM-head events of an armed step are given to entmtp_step_arm");
    st->armed = false;
    open_gate(st);
    lm_ready = T <= st->armed_T && hidden == st->armed_hidden && w_step == st->armed_w;
    st->lm_parts = st->armed_parts;
  } else {
    // the side stream's work of this step starts after everything the
    // caller enqueued before it (the step's inputs)
    if (int32_t rc = hip_status(hipEventRecord(st->fork, s), "hipEventRecord (fork)")) return rc;
  }

  if (!lm_ready) {
    // a timed LM head waits behind a launch gate that opens once it is enqueued
    const bool gated = ev_lm_begin != nullptr;
    if (gated)
      if (int32_t rc = enqueue_gate(st, s)) return rc;
    // the LM head (the longest kernel) is enqueued first, so that it is
    // running while the host enqueues the attention chain behind it
    const int32_t lm_rc = launch_step_partials(
        hidden, static_cast<const entmtp_bf16*>(w_step), T, c.hid, c.V, c.inv_temp, c.logits, part,
        &st->lm_parts, s, static_cast<hipEvent_t>(ev_lm_begin), static_cast<hipEvent_t>(ev_lm_end));
    if (gated) open_gate(st);
    if (lm_rc) return lm_rc;
  }
  // the statistics merge and acceptance wait for the LM head: with one layer
  // they are enqueued after the short attention chain (which then starts a
  // few microseconds sooner), with many before it (whose enqueue would
  // outlast the LM head)
  const uint32_t seq = st->seq + 1u == 0u ? 1u : st->seq + 1u;   // 0 is the record's initial tag
  auto finalize = [&]() {
    return launch_finalize_accept(st->bank, topo, part, st->lm_parts, c.V, c.inv_temp, c.entropy,
                                  c.top1p, c.argmax, draft_tokens, c.accept_len, c.path,
                                  c.path_capacity, c.bonus, c.best_top1p, st->dev, seq, s);
  };
  if (c.n_layers > 1)
    if (int32_t rc = finalize()) return rc;
  // the cache chain on the side stream, concurrent with the LM head: the
  // previous step's compaction, then this step's attention layers
  if (int32_t rc = hip_status(hipStreamWaitEvent(st->side, st->fork, 0), "hipStreamWaitEvent"))
    return rc;
  if (int32_t rc = enqueue_due_compaction(st)) return rc;
  const size_t q_layer = static_cast<size_t>(c.tree_rows) * c.Hq * c.d;
  const size_t kv_layer = static_cast<size_t>(c.tree_rows) * c.Hkv * c.d;
  for (int32_t l = 0; l < c.n_layers; ++l) {
    const size_t cl = static_cast<size_t>(l) * static_cast<size_t>(c.cache_layer_stride);
    if (int32_t rc = entmtp_tree_attn(st->bank, topo, q + l * q_layer, k_tree + l * kv_layer,
                                      v_tree + l * kv_layer, c.k_cache + cl, c.v_cache + cl, c.cap,
                                      prefix_len, c.Hq, c.Hkv, c.d, c.scale, c.rope_theta,
                                      out + l * q_layer, ws, st->attn_bytes, st->side))
      return rc;
  }
  if (c.n_layers == 1)
    if (int32_t rc = finalize()) return rc;
  st->seq = seq;
  st->pending = true;
  st->pending_L = prefix_len;
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_step_arm(entmtp_step* st, const entmtp_bf16* hidden,
                                   const entmtp_bf16* w_lm, int32_t T_bound, void* ev_lm_begin,
                                   void* ev_lm_end) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr, ENTMTP_EINVAL, "step is NULL");
  ENTMTP_CHECK_ARG(!st->armed, ENTMTP_EINVAL, "the next step is armed already");
  ENTMTP_CHECK_ARG(!st->dev_started, ENTMTP_EINVAL,
                   "device-scheduled steps are running (their LM heads are enqueued by their launch)");
  ENTMTP_CHECK_ARG(hidden != nullptr, ENTMTP_EINVAL, "hidden is NULL");
  ENTMTP_CHECK_ARG(w_lm == nullptr || aligned16(w_lm), ENTMTP_EINVAL, "w_lm must be 16-byte aligned");
  ENTMTP_CHECK_ARG(T_bound >= 1 && T_bound <= st->T_max, ENTMTP_ERANGE,
                   "T_bound = %d outside [1, %d] (the bank's largest tree)", T_bound, st->T_max);
  const entmtp_step_config& c = st->cfg;
  auto s = static_cast<hipStream_t>(c.stream);
  void* part = static_cast<uint8_t*>(c.workspace) + st->part_offset;
  const void* w_step = w_lm ? w_lm : c.w_lm;
  // the next step's cache chain starts after everything enqueued so far (the
  // caller's inputs and the pending step's acceptance), not after the armed
  // LM head
  if (int32_t rc = hip_status(hipEventRecord(st->fork, s), "hipEventRecord (fork)")) return rc;
  if (int32_t rc = enqueue_gate(st, s)) return rc;
  int32_t parts = 0;
  const int32_t rc = launch_step_partials(
      hidden, static_cast<const entmtp_bf16*>(w_step), T_bound, c.hid, c.V, c.inv_temp, c.logits,
      part, &parts, s, static_cast<hipEvent_t>(ev_lm_begin), static_cast<hipEvent_t>(ev_lm_end));
  if (rc) {
    open_gate(st);
    return rc;
  }
  st->armed = true;
  st->armed_T = T_bound;
  st->armed_parts = parts;
  st->armed_hidden = hidden;
  st->armed_w = w_step;
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_step_wait(entmtp_step* st, int32_t* accept_len, int32_t* bonus,
                                    float* best_top1p, double timeout_s) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr, ENTMTP_EINVAL, "step is NULL");
  ENTMTP_CHECK_ARG(st->pending, ENTMTP_EINVAL, "no launched step is waiting to be read");
  ENTMTP_CHECK_ARG(timeout_s >= 0.0, ENTMTP_EINVAL, "timeout_s must be >= 0");
  const uint32_t want = st->seq;
  const auto t0 = std::chrono::steady_clock::now();
  auto s = static_cast<hipStream_t>(st->cfg.stream);
  const uint64_t* words = reinterpret_cast<const uint64_t*>(st->host);
  // the record is complete once every word it needs carries the sequence number
  auto complete = [&]() {
    const uint64_t w0 = __atomic_load_n(&words[0], __ATOMIC_ACQUIRE);
    if (static_cast<uint32_t>(w0 >> 32) != want) return false;
    const int a = static_cast<int32_t>(static_cast<uint32_t>(w0));
    const int n = 3 + (a < 0 || a > ENTMTP_D_MAX ? kMirrorPathWords : a / 4 + 1);
    for (int k = 1; k < n; ++k)
      if (static_cast<uint32_t>(__atomic_load_n(&words[k], __ATOMIC_ACQUIRE) >> 32) != want)
        return false;
    return true;
  };
  for (uint32_t spin = 1;; ++spin) {
    if (complete()) break;
    if ((spin & 255u) == 0u) {
      // every few hundred polls: a failed stream or an expired limit ends the wait
      const hipError_t e = hipStreamQuery(s);
      if (e == hipSuccess) {
        if (complete()) break;
        st->pending = false;
        return fail(ENTMTP_EHIP, "stream idle but step %u published no result", want);
      }
      if (e != hipErrorNotReady) {
        st->pending = false;
        return hip_status(e, "stream error while waiting for the step");
      }
      const double el = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
      if (el > timeout_s)
        return fail(ENTMTP_ETIMEDOUT, "no result for step %u after %.3f s", want, el);
    }
    __builtin_ia32_pause();
  }
  // the result is known: an armed LM head (sized for any tree the caller may
  // choose next) may start now, before the caller has moved the ladder
  if (st->armed) open_gate(st);
  const int32_t a = static_cast<int32_t>(static_cast<uint32_t>(words[0]));
  st->pending = false;
  if (a < 0 || a > st->D_max)
    return fail(ENTMTP_EHIP, "step %u published accept length %d outside [0, %d]", want, a,
                st->D_max);
  if (accept_len) *accept_len = a;
  if (bonus) *bonus = static_cast<int32_t>(static_cast<uint32_t>(words[1]));
  if (best_top1p) {
    const uint32_t bits = static_cast<uint32_t>(words[2]);
    std::memcpy(best_top1p, &bits, sizeof(float));
  }
  // the path for this step's compaction, which the next launch (or a flush) enqueues
  for (int j = 0; j <= a; ++j)
    st->due_path[j] = static_cast<int32_t>((words[3 + j / 4] >> (8 * (j % 4))) & 0xffu);
  st->due_a = a;
  st->due_L = st->pending_L;
  st->compact_due = true;
  return ENTMTP_OK;
}

namespace {

__global__ void device_start_kernel(DevStep* state, const DevTopo* topos, int rung, int L) {
  if (threadIdx.x == 0) state[0] = DevStep{rung, topos[rung].T, L, 0, 0};
}

}  // namespace

extern "C" int32_t entmtp_step_device_start(entmtp_step* st, int32_t topo, int32_t prefix_len) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr, ENTMTP_EINVAL, "step is NULL");
  if (int32_t rc = check_device_bank(st->bank, topo)) return rc;
  const entmtp_step_config& c = st->cfg;
  ENTMTP_CHECK_ARG(prefix_len >= 0 && static_cast<int64_t>(prefix_len) + st->bank->desc[topo].T <= c.cap,
                   ENTMTP_ERANGE, "prefix_len %d + T %d outside the cache capacity %d", prefix_len,
                   st->bank->desc[topo].T, c.cap);
  ENTMTP_CHECK_ARG(st->T_max <= 128, ENTMTP_ERANGE,
                   "device-scheduled steps support trees of up to 128 nodes (bank has %d)", st->T_max);
  // steps before this one finish their cache work first (an armed LM head
  // runs unused: device-scheduled steps enqueue their own)
  if (int32_t rc = flush_side(st)) return rc;
  st->armed = false;
  DevStep* state = dev_state(st);
  hipLaunchKernelGGL(device_start_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(c.stream),
                     state, reinterpret_cast<const DevTopo*>(state + entmtp_step::kRing), topo,
                     prefix_len);
  if (int32_t rc = launch_status("device_start launch")) return rc;
  st->dev_started = true;
  st->dev_t = 0;
  st->dev_compact = 0;
  st->dev_sync_t = 0;
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_step_launch_device(entmtp_step* st, const entmtp_bf16* q,
                                             const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                                             entmtp_bf16* out, const entmtp_bf16* hidden,
                                             const entmtp_bf16* w_lm, const int32_t* drafts,
                                             int32_t* log, int32_t log_rows, void* ev_lm_begin,
                                             void* ev_lm_end) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr, ENTMTP_EINVAL, "step is NULL");
  ENTMTP_CHECK_ARG(st->dev_started, ENTMTP_EINVAL, "entmtp_step_device_start was not called");
  ENTMTP_CHECK_ARG(q && k_tree && v_tree && out && hidden && drafts, ENTMTP_EINVAL,
                   "per-step inputs and outputs must be non-NULL");
  ENTMTP_CHECK_ARG(log == nullptr || log_rows >= 1, ENTMTP_EINVAL, "log_rows = %d < 1", log_rows);
  ENTMTP_CHECK_ARG(w_lm == nullptr || aligned16(w_lm), ENTMTP_EINVAL, "w_lm must be 16-byte aligned");
  const entmtp_step_config& c = st->cfg;
  auto s = static_cast<hipStream_t>(c.stream);
  uint8_t* ws = static_cast<uint8_t*>(c.workspace);
  void* part = ws + st->part_offset;
  constexpr int R = entmtp_step::kRing;
  const uint64_t t = st->dev_t;
  DevStep* state = dev_state(st);
  const auto* topos = reinterpret_cast<const DevTopo*>(state + R);
  DevStep* cur = state + t % R;
  DevStep* next = state + (t + 1) % R;
  int32_t* ring = dev_ring(st, t);

  // the cache chain starts after everything the caller enqueued so far: the
  // previous step's acceptance (this step's tree and prefix length) and this
  // step's inputs
  if (int32_t rc = hip_status(hipEventRecord(st->fork, s), "hipEventRecord (fork)")) return rc;

  // the caller's stream: LM head, then statistics + acceptance + ladder
  if (int32_t rc = launch_partials_device_T(hidden, w_lm ? w_lm : c.w_lm, &cur->T, st->T_max, c.hid,
                                            c.V, c.inv_temp, part, s,
                                            static_cast<hipEvent_t>(ev_lm_begin),
                                            static_cast<hipEvent_t>(ev_lm_end)))
    return rc;
  // step t writes state slot t+1 and ring slot t, which the side stream's
  // work of step t+2-R read last: one wait for its step t-kWaitLag every
  // kWaitEvery steps covers that (steps whose side work a flush has joined
  // need none)
  constexpr uint64_t E = entmtp_step::kWaitEvery, LAG = entmtp_step::kWaitLag;
  if (t % E == 0 && t >= st->dev_sync_t + LAG)
    if (int32_t rc = hip_status(hipStreamWaitEvent(s, st->ev_side[(t - LAG) % R], 0),
                                "hipStreamWaitEvent"))
      return rc;
  FinAccDevice dv;
  dv.cur = cur;
  dv.next = next;
  dv.topos = topos;
  dv.drafts = drafts;
  dv.tree_rows = c.tree_rows;
  dv.n_topo = static_cast<int32_t>(st->bank->desc.size());
  dv.cap = c.cap;
  dv.prefix_fixed = c.device_prefix_fixed;
  dv.tau_on = c.tau_on;
  dv.tau_off = c.tau_off;
  dv.log = log;
  dv.log_rows = log_rows;
  dv.user_accept_len = c.accept_len;
  dv.user_path = c.path;
  if (int32_t rc = launch_finalize_accept_device(st->bank, dv, part, c.V, c.inv_temp, c.entropy,
                                                 c.top1p, c.argmax, ring, ring + 1,
                                                 c.path_capacity, c.bonus, c.best_top1p, nullptr,
                                                 0u, s))
    return rc;

  // the side stream: the previous step's compaction, then this step's attention
  if (int32_t rc = hip_status(hipStreamWaitEvent(st->side, st->fork, 0), "hipStreamWaitEvent"))
    return rc;
  if (t >= 1 && st->dev_compact < t)
    if (int32_t rc = enqueue_device_compaction(st, t - 1)) return rc;
  const size_t q_layer = static_cast<size_t>(c.tree_rows) * c.Hq * c.d;
  const size_t kv_layer = static_cast<size_t>(c.tree_rows) * c.Hkv * c.d;
  for (int32_t l = 0; l < c.n_layers; ++l) {
    const size_t cl = static_cast<size_t>(l) * static_cast<size_t>(c.cache_layer_stride);
    if (int32_t rc = launch_attn_device(st->bank, cur, topos, st->dshape, q + l * q_layer,
                                        k_tree + l * kv_layer, v_tree + l * kv_layer,
                                        c.k_cache + cl, c.v_cache + cl, c.cap, c.Hq, c.Hkv,
                                        c.scale, c.rope_theta, out + l * q_layer, ws, st->side))
      return rc;
  }
  if (int32_t rc = hip_status(hipEventRecord(st->ev_side[t % R], st->side), "hipEventRecord"))
    return rc;
  st->dev_t = t + 1;
  return ENTMTP_OK;
}

namespace {

// A captured segment and the ring slot its first step reads (the device
// state must sit in that slot when the segment is replayed).
struct StepGraph {
  hipGraphExec_t exec;
  int slot;
};

}  // namespace

extern "C" int32_t entmtp_step_device_graph(entmtp_step* st, int32_t n_steps,
                                            const entmtp_bf16* const* q,
                                            const entmtp_bf16* const* k_tree,
                                            const entmtp_bf16* const* v_tree,
                                            entmtp_bf16* const* out,
                                            const entmtp_bf16* const* hidden,
                                            const entmtp_bf16* const* w_lm,
                                            const int32_t* const* drafts, int32_t* log,
                                            int32_t log_rows, void** graph) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr && graph != nullptr, ENTMTP_EINVAL, "step or graph is NULL");
  *graph = nullptr;
  ENTMTP_CHECK_ARG(st->dev_started, ENTMTP_EINVAL, "entmtp_step_device_start was not called");
  ENTMTP_CHECK_ARG(n_steps >= entmtp_step::kRing && n_steps % entmtp_step::kRing == 0,
                   ENTMTP_EINVAL, "n_steps = %d must be a positive multiple of %d", n_steps,
                   entmtp_step::kRing);
  ENTMTP_CHECK_ARG(q && k_tree && v_tree && out && hidden && drafts, ENTMTP_EINVAL,
                   "per-step pointer arrays must be non-NULL host arrays");
  ENTMTP_CHECK_ARG(st->cfg.stream != nullptr, ENTMTP_EINVAL,
                   "capturing needs a created stream (not the null stream)");
  auto s = static_cast<hipStream_t>(st->cfg.stream);
  // the segment starts from a joined state, so it depends on nothing outside it
  if (int32_t rc = flush_side(st)) return rc;
  const int slot = static_cast<int>(st->dev_t % entmtp_step::kRing);
  if (int32_t rc = hip_status(hipStreamBeginCapture(s, hipStreamCaptureModeRelaxed),
                              "hipStreamBeginCapture"))
    return rc;
  int32_t rc = ENTMTP_OK;
  for (int32_t i = 0; i < n_steps && rc == ENTMTP_OK; ++i)
    rc = entmtp_step_launch_device(st, q[i], k_tree[i], v_tree[i], out[i], hidden[i],
                                   w_lm ? w_lm[i] : nullptr, drafts[i], log, log_rows, nullptr,
                                   nullptr);
  if (rc == ENTMTP_OK) rc = flush_side(st);   // ... and ends joined
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(s, &g);
  if (rc == ENTMTP_OK) rc = hip_status(e, "hipStreamEndCapture");
  hipGraphExec_t exec = nullptr;
  if (rc == ENTMTP_OK)
    rc = hip_status(hipGraphInstantiate(&exec, g, nullptr, nullptr, 0), "hipGraphInstantiate");
  if (g) (void)hipGraphDestroy(g);
  if (rc != ENTMTP_OK) return rc;
  *graph = new StepGraph{exec, slot};
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_step_graph_launch(entmtp_step* st, void* graph) {
  clear_error();
  ENTMTP_CHECK_ARG(st != nullptr && graph != nullptr, ENTMTP_EINVAL, "step or graph is NULL");
  const auto* g = static_cast<const StepGraph*>(graph);
  const int now = static_cast<int>(st->dev_t % entmtp_step::kRing);
  ENTMTP_CHECK_ARG(now == g->slot, ENTMTP_EINVAL,
                   "the device state is in ring slot %d, the segment starts at slot %d: eager "
                   "steps between replays must number a multiple of %d", now, g->slot,
                   entmtp_step::kRing);
  return hip_status(hipGraphLaunch(g->exec, static_cast<hipStream_t>(st->cfg.stream)),
                    "hipGraphLaunch");
}

extern "C" void entmtp_step_graph_destroy(void* graph) {
  if (!graph) return;
  auto* g = static_cast<StepGraph*>(graph);
  (void)hipGraphExecDestroy(g->exec);
  delete g;
}
