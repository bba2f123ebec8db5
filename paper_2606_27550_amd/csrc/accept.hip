// Greedy tree acceptance and the longest accepted path.
//
// Left-to-right acceptance of §2.1, in its greedy form over a tree: a node is
// accepted when its draft token equals the target's greedy token at its
// parent and every ancestor is accepted.  With the tree's ancestor bitmask
// (the same per-node rows the attention kernel uses) "every ancestor is
// accepted" becomes a subset test of the node's mask row against the set of
// locally matching nodes, so all nodes are decided in parallel.  The answer is
// the deepest accepted node, lowest index among equals; its depth is the
// accept length (§5.1).  One workgroup handles the whole tree.  Inside a
// verification step of a small tree the acceptance runs fused behind the
// statistics in one workgroup: its wavefronts merge the LM head's partials
// node by node into LDS, and the same workgroup then accepts the tree from
// there, so no device-wide fence or arrival counter sits between the two.
// Larger trees merge their statistics in a kernel of their own, one
// wavefront per node, before the acceptance kernel.
#include "accept.hpp"
#include "common.hpp"
#include "stats.hpp"

namespace entmtp {
namespace {

// statistics + acceptance of one step, one workgroup: sixteen wavefronts, so
// that each merges one node's partials per pass (a wavefront merging eight
// nodes at once ran a chain eight times as long: 10 us against 6 us for the
// 27-node tree)
constexpr int kFinAccThreads = 1024;
constexpr int kPathPerThread = 1;       // path-table entries a thread carries across the merge
constexpr int kFusedMaxT = 32;         // larger trees: a separate statistics kernel



__device__ __forceinline__ void accept_core(
    const int* __restrict__ parent, const int* __restrict__ depth,
    const uint32_t* __restrict__ mask, const int* __restrict__ path_tab, int T, int D,
    const int* __restrict__ tok, const int* __restrict__ amax, const float* __restrict__ top1p,
    int* __restrict__ accept_len, int* __restrict__ path_out, int path_cap,
    int* __restrict__ bonus, float* __restrict__ best_p, StepMirror* __restrict__ mirror,
    uint32_t seq) {
  const NodeIn n = accept_load(parent, depth, mask, tok, T);
  (void)accept_finish(n, greedy_ok(n, amax, T), path_tab, T, D, amax, top1p, accept_len, path_out,
                      path_cap, bonus, best_p, mirror, seq);
}

__global__ __launch_bounds__(kAcceptThreads) void accept_kernel(
    const int* __restrict__ parent, const int* __restrict__ depth,
    const uint32_t* __restrict__ mask, const int* __restrict__ path_tab, int T, int D,
    const int* __restrict__ tok, const int* __restrict__ amax, const float* __restrict__ top1p,
    int* __restrict__ accept_len, int* __restrict__ path_out, int path_cap,
    int* __restrict__ bonus, float* __restrict__ best_p, StepMirror* __restrict__ mirror,
    uint32_t seq) {
  accept_core(parent, depth, mask, path_tab, T, D, tok, amax, top1p, accept_len, path_out, path_cap,
              bonus, best_p, mirror, seq);
}

// One tree of a batch: its bank arrays and its rows in the concatenated
// per-node arrays.
struct AcceptSeq {
  const int* parent;
  const int* depth;
  const uint32_t* mask;
  const int* path_tab;
  int T, D, row0;
};

struct AcceptBatch {
  AcceptSeq s[ENTMTP_B_MAX];
  const int* tok;
  const int* amax;
  const float* top1p;
  int* accept_len;
  int* path;
  int path_cap;
  int* bonus;
  float* best;
};

// Workgroup b accepts tree b.
__global__ __launch_bounds__(kAcceptThreads) void accept_batched_kernel(AcceptBatch p) {
  const int b = blockIdx.x;
  const AcceptSeq& q = p.s[b];
  accept_core(q.parent, q.depth, q.mask, q.path_tab, q.T, q.D, p.tok + q.row0, p.amax + q.row0,
              p.top1p ? p.top1p + q.row0 : nullptr, p.accept_len + b,
              p.path + static_cast<size_t>(b) * p.path_cap, p.path_cap, p.bonus + b,
              p.best ? p.best + b : nullptr, nullptr, 0u);
}

// A batch whose trees and rows are device arrays (topo[b], row_off[b]):
// every bank tree's arrays travel in the kernel arguments.
constexpr int kMaxTreesAccept = 32;
struct AcceptBatchDev {
  AcceptSeq trees[kMaxTreesAccept];   // row0 unused
  const int* topo;
  const int* row_off;                 // [B + 1]
  int rows_cap, n_trees;
  const int* tok;
  const int* amax;
  const float* top1p;
  int* accept_len;
  int* path;
  int path_cap;
  int* bonus;
  float* best;
};

static_assert(sizeof(AcceptBatchDev) <= 4096, "kernel arguments are limited to 4 KB");

// Workgroup b accepts sequence b's tree.  A sequence whose tree index lies
// outside the bank, whose tree rows [row_off[b], row_off[b] + T) do not lie
// in [row_off[b], row_off[b + 1]) and the row capacity, or whose tree is
// deeper than the path rows hold is not verified: accept length -1, path and
// bonus -1 (compaction then moves nothing).
__global__ __launch_bounds__(kAcceptThreads) void accept_batched_device_kernel(AcceptBatchDev p) {
  const int b = blockIdx.x;
  const int tr = p.topo[b], r0 = p.row_off[b], r1 = p.row_off[b + 1];
  const bool named = tr >= 0 && tr < p.n_trees;
  const int T = p.trees[named ? tr : 0].T;
  const long long end = static_cast<long long>(r0) + T;   // (64-bit: the entries are unchecked)
  const bool ok = named && r0 >= 0 && end <= r1 && end <= p.rows_cap &&
                  p.trees[named ? tr : 0].D + 1 <= p.path_cap;
  int* path = p.path + static_cast<size_t>(b) * p.path_cap;
  if (!ok) {
    for (int i = threadIdx.x; i < p.path_cap; i += blockDim.x) path[i] = -1;
    if (threadIdx.x == 0) {
      p.accept_len[b] = -1;
      p.bonus[b] = -1;
      if (p.best) p.best[b] = 0.f;
    }
    return;
  }
  const AcceptSeq& q = p.trees[tr];
  accept_core(q.parent, q.depth, q.mask, q.path_tab, q.T, q.D, p.tok + r0, p.amax + r0,
              p.top1p ? p.top1p + r0 : nullptr, p.accept_len + b, path, p.path_cap, p.bonus + b,
              p.best ? p.best + b : nullptr, nullptr, 0u);
}

// Statistics of every node of the tree from the LM head's partials, then the
// acceptance of the tree, by one workgroup of kFinAccThreads threads.
__global__ __launch_bounds__(kFinAccThreads) void finalize_accept_kernel(
    const StatPart* __restrict__ part, int G, float inv_temp, float* __restrict__ entropy,
    float* __restrict__ top1p, int* __restrict__ amax, const int* __restrict__ parent,
    const int* __restrict__ depth, const uint32_t* __restrict__ mask,
    const int* __restrict__ path_tab, int T, int D, const int* __restrict__ tok,
    int* __restrict__ accept_len, int* __restrict__ path_out, int path_cap,
    int* __restrict__ bonus, float* __restrict__ best_p, StepMirror* __restrict__ mirror,
    uint32_t seq) {
  constexpr int kPathLds = kPathPerThread * kFinAccThreads;
  __shared__ float s_p1[ENTMTP_T_MAX];
  __shared__ int s_am[ENTMTP_T_MAX];
  __shared__ int s_path[kPathLds];
  // the tree's own inputs, and its path table when it fits in LDS, are
  // fetched while the partials merge (the path rows are then read from LDS
  // at the end instead of by a dependent global load)
  const NodeIn n = accept_load(parent, depth, mask, tok, T);
  const int np = T * (D + 1);
  const bool lds_path = np <= kPathLds;
  int pv[kPathPerThread];
#pragma unroll
  for (int k = 0; k < kPathPerThread; ++k) {
    const int idx = threadIdx.x + k * kFinAccThreads;
    pv[k] = lds_path && idx < np ? path_tab[idx] : -1;
  }
  // up to 32 nodes merge in one pass (eight rows per wavefront) when the LM
  // head folded two slices per partial
  finalize_nodes<kFinAccThreads>(part, G, T, inv_temp, entropy, top1p, amax, s_p1, s_am);
  if (lds_path) {
#pragma unroll
    for (int k = 0; k < kPathPerThread; ++k) {
      const int idx = threadIdx.x + k * kFinAccThreads;
      if (idx < np) s_path[idx] = pv[k];
    }
  }
  __syncthreads();
  (void)accept_finish<kFinAccThreads>(n, greedy_ok(n, s_am, T), lds_path ? s_path : path_tab, T,
                                      D, s_am, s_p1, accept_len, path_out, path_cap, bonus,
                                      best_p, mirror, seq);
}

// The same for a tree the device chose: the tree, its drafts and the prefix
// length come from *dv.cur; the workgroup also runs the ladder and writes the
// next step's state (tree, node count, prefix length).
constexpr int kFinAccDevThreads = 1024;   // any bank tree (up to 128 nodes) in at most 4 passes
__global__ __launch_bounds__(kFinAccDevThreads) void finalize_accept_device_kernel(
    FinAccDevice dv, const uint8_t* __restrict__ arena, const StatPart* __restrict__ part, int G,
    int G_small, float inv_temp, float* __restrict__ entropy, float* __restrict__ top1p,
    int* __restrict__ amax, int* __restrict__ accept_len, int* __restrict__ path_out,
    int path_cap, int* __restrict__ bonus, float* __restrict__ best_p,
    StepMirror* __restrict__ mirror, uint32_t seq) {
  __shared__ float s_p1[ENTMTP_T_MAX];
  __shared__ int s_am[ENTMTP_T_MAX];
  const DevStep st = *dv.cur;
  const int T = st.T;
  const DevTopo* t = dv.topos + st.rung;
  const int* parent = reinterpret_cast<const int*>(arena + t->off_parent);
  const int* depth = reinterpret_cast<const int*>(arena + t->off_depth);
  const uint32_t* mask = reinterpret_cast<const uint32_t*>(arena + t->off_mask);
  const int* path_tab = reinterpret_cast<const int*>(arena + t->off_path);
  const int D = t->D;
  const int* tok = dv.drafts + static_cast<size_t>(st.rung) * dv.tree_rows;
  const NodeIn n = accept_load(parent, depth, mask, tok, T);
  // the small-tree LM head wrote one partial per workgroup (G_small per row)
  finalize_nodes<kFinAccDevThreads>(part, T <= kStepSmallT ? G_small : G, T, inv_temp, entropy,
                                    top1p, amax, s_p1, s_am);
  __syncthreads();
  const int key = accept_finish<kFinAccDevThreads>(n, greedy_ok(n, s_am, T), path_tab, T, D, s_am,
                                                   s_p1, accept_len, path_out, path_cap, bonus,
                                                   best_p, mirror, seq);
  {
    const int i = threadIdx.x, a = key >> 10, best = 1023 - (key & 1023);
    if (dv.user_path && i < path_cap) dv.user_path[i] = i <= a ? path_tab[best * (D + 1) + i] : -1;
    if (dv.user_accept_len && i == 0) *dv.user_accept_len = a;
  }
  if (threadIdx.x == 0) {
    const int a = key >> 10, best = 1023 - (key & 1023);
    const float s = s_p1[best];
    // a step beyond the cache verified nothing: stop where it is
    const bool over = st.overflow != 0 || st.L + st.T > dv.cap;
    const int next = over ? st.rung : ladder_step(st.rung, dv.n_topo, s, dv.tau_on, dv.tau_off);
    DevStep nx;
    nx.rung = next;
    nx.T = dv.topos[next].T;
    nx.L = over || dv.prefix_fixed ? st.L : st.L + a + 1;
    nx.step = st.step + 1;
    nx.overflow = over ? 1 : 0;
    *dv.next = nx;
    if (dv.log) {
      int32_t* row = dv.log + 4 * static_cast<size_t>(st.step % dv.log_rows);
      row[0] = st.rung;
      row[1] = st.L;
      row[2] = over ? -1 : a;
      row[3] = __float_as_int(s);
    }
  }
}

// Logits of node i's draft token and of its parent's argmax under the
// parent's LM-head row: X[parent] . W[tok] and X[parent] . W[argmax[parent]]
// (fp32), one wave per node.  A draft token outside [0, V) gets -inf.
__global__ __launch_bounds__(64) void draft_logits_kernel(
    const int* __restrict__ parent, const uint16_t* __restrict__ X,
    const uint16_t* __restrict__ W, int hid, int V, const int* __restrict__ tok,
    const int* __restrict__ amax, float* __restrict__ z_draft, float* __restrict__ z_top) {
  const int i = blockIdx.x, lane = threadIdx.x;
  if (i == 0) {
    if (lane == 0) {
      z_draft[0] = 0.f;
      z_top[0] = 0.f;
    }
    return;
  }
  const int p = parent[i];
  const int t = tok[i];
  const bool valid = t >= 0 && t < V;
  int a = amax[p];
  a = a < 0 ? 0 : (a >= V ? V - 1 : a);
  const uint16_t* x = X + static_cast<size_t>(p) * hid;
  const uint16_t* w1 = W + static_cast<size_t>(valid ? t : 0) * hid;
  const uint16_t* w2 = W + static_cast<size_t>(a) * hid;
  float s1 = 0.f, s2 = 0.f;
  for (int c = lane; c < hid / 8; c += 64) {
    const u32x4 xv = *reinterpret_cast<const u32x4*>(x + 8 * c);
    const u32x4 v1 = *reinterpret_cast<const u32x4*>(w1 + 8 * c);
    const u32x4 v2 = *reinterpret_cast<const u32x4*>(w2 + 8 * c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float xl = __uint_as_float(xv[e] << 16), xh = __uint_as_float(xv[e] & 0xFFFF0000u);
      s1 += xl * __uint_as_float(v1[e] << 16) + xh * __uint_as_float(v1[e] & 0xFFFF0000u);
      s2 += xl * __uint_as_float(v2[e] << 16) + xh * __uint_as_float(v2[e] & 0xFFFF0000u);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    s1 += __shfl_xor(s1, off, 64);
    s2 += __shfl_xor(s2, off, 64);
  }
  if (lane == 0) {
    z_draft[i] = valid ? s1 : -INFINITY;
    z_top[i] = s2;
  }
}

// Typical acceptance: node i >= 1 is locally acceptable when its draft
// token's probability under the parent's temperature-scaled distribution,
// p_i = exp((z_draft - z_top) * inv_temp) * top1p[parent], exceeds
// min(eps, alpha * exp(-entropy[parent])).  Among the deepest accepted nodes
// the one whose path's drafts are jointly most likely wins (largest sum of
// log p over its root-to-node path, then the lowest index): under this rule
// several siblings often pass together.  The key packs depth (5 bits), the
// order-preserving bits of that fp32 sum and 1023 - index into 64 bits, so
// one maximum over the workgroup makes the choice.
__device__ __forceinline__ uint64_t float_order_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__global__ __launch_bounds__(kAcceptThreads) void accept_typical_kernel(
    const int* __restrict__ parent, const int* __restrict__ depth,
    const uint32_t* __restrict__ mask, const int* __restrict__ path_tab, int T, int D,
    const int* __restrict__ tok, const int* __restrict__ amax, const float* __restrict__ z_draft,
    const float* __restrict__ z_top, const float* __restrict__ entropy,
    const float* __restrict__ top1p, float inv_temp, float eps, float alpha,
    int* __restrict__ accept_len, int* __restrict__ path_out, int* __restrict__ bonus,
    float* __restrict__ best_p) {
  __shared__ float s_logp[kAcceptThreads];
  __shared__ uint32_t matched[ENTMTP_MASK_WORDS];
  __shared__ uint64_t s_key[kAcceptThreads / 64];
  const NodeIn n = accept_load(parent, depth, mask, tok, T);
  const int i = threadIdx.x;
  bool ok = false;
  float logp = 0.f;
  if (i == 0) {
    ok = true;
  } else if (i < T) {
    const int p = n.parent;
    const float pd = expf((z_draft[i] - z_top[i]) * inv_temp) * top1p[p];
    const float thr = fminf(eps, alpha * expf(-entropy[p]));
    ok = pd > thr;
    logp = ok ? logf(pd) : 0.f;   // pd > thr >= 0 for every node whose value is read
  }
  s_logp[i] = logp;
  if (i < ENTMTP_MASK_WORDS) matched[i] = 0u;
  __syncthreads();
  if (i < T && ok) atomicOr(&matched[i >> 5], 1u << (i & 31));
  __syncthreads();
  uint64_t key = 0u;   // below every accepted node's key (the root's is > 0)
  if (i < T) {
    bool acc = true;
#pragma unroll
    for (int w = 0; w < ENTMTP_MASK_WORDS; ++w) acc = acc && ((n.mask[w] & ~matched[w]) == 0u);
    if (acc) {
      float ll = 0.f;   // root to node, as the path is walked
      for (int j = 1; j <= n.depth; ++j) ll += s_logp[path_tab[i * (D + 1) + j]];
      key = (static_cast<uint64_t>(n.depth) << 42) | (float_order_bits(ll) << 10) |
            static_cast<uint64_t>(1023 - i);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(key), off, 64);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(key >> 32), off, 64);
    const uint64_t other = (static_cast<uint64_t>(hi) << 32) | lo;
    key = other > key ? other : key;
  }
  if ((i & 63) == 0) s_key[i >> 6] = key;
  __syncthreads();
  key = s_key[0];
#pragma unroll
  for (int w = 1; w < kAcceptThreads / 64; ++w) key = s_key[w] > key ? s_key[w] : key;
  const int best = 1023 - static_cast<int>(key & 1023u);
  const int a = static_cast<int>(key >> 42);
  if (i <= D) path_out[i] = (i <= a) ? path_tab[best * (D + 1) + i] : -1;
  if (i == 0) {
    *accept_len = a;
    *bonus = amax[best];
    if (best_p) *best_p = top1p[best];
  }
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

namespace entmtp {

int32_t launch_accept(const entmtp_bank* bank, int32_t topo, const int32_t* draft_tokens,
                      const int32_t* argmax, const float* top1p, int32_t* accept_len,
                      int32_t* path, int32_t path_capacity, int32_t* bonus, float* best_top1p,
                      StepMirror* mirror, uint32_t seq, hipStream_t stream) {
  const TopoDesc& d = bank->desc[topo];
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(kAcceptThreads), 0, stream,
                     bank_ptr<int>(bank, d.off_parent), bank_ptr<int>(bank, d.off_depth),
                     bank_ptr<uint32_t>(bank, d.off_mask), bank_ptr<int>(bank, d.off_path), d.T,
                     d.D, draft_tokens, argmax, top1p, accept_len, path, path_capacity, bonus,
                     best_top1p, mirror, seq);
  return launch_status("accept launch");
}

int32_t launch_finalize_accept_device(const entmtp_bank* bank, const FinAccDevice& dv,
                                      const void* partials, int32_t V, float inv_temp,
                                      float* entropy, float* top1p, int32_t* argmax,
                                      int32_t* accept_len, int32_t* path, int32_t path_capacity,
                                      int32_t* bonus, float* best_top1p, StepMirror* mirror,
                                      uint32_t seq, hipStream_t stream) {
  hipLaunchKernelGGL(finalize_accept_device_kernel, dim3(1), dim3(kFinAccDevThreads), 0, stream, dv,
                     bank->arena, static_cast<const StatPart*>(partials), stats_slices(V),
                     step_small_parts(V), inv_temp, entropy, top1p, argmax, accept_len, path, path_capacity, bonus,
                     best_top1p, mirror, seq);
  return launch_status("finalize_accept (device-scheduled) launch");
}

int32_t launch_finalize_accept(const entmtp_bank* bank, int32_t topo, const void* partials,
                               int32_t n_parts, int32_t V, float inv_temp, float* entropy,
                               float* top1p,
                               int32_t* argmax, const int32_t* draft_tokens, int32_t* accept_len,
                               int32_t* path, int32_t path_capacity, int32_t* bonus,
                               float* best_top1p, StepMirror* mirror, uint32_t seq,
                               hipStream_t stream) {
  const TopoDesc& d = bank->desc[topo];
  if (d.T > kFusedMaxT) {
    if (int32_t rc = launch_stats_finalize(partials, d.T, V, inv_temp, entropy, top1p, argmax, stream))
      return rc;
    return launch_accept(bank, topo, draft_tokens, argmax, top1p, accept_len, path, path_capacity,
                         bonus, best_top1p, mirror, seq, stream);
  }
  hipLaunchKernelGGL(finalize_accept_kernel, dim3(1), dim3(kFinAccThreads), 0, stream,
                     static_cast<const StatPart*>(partials), n_parts, inv_temp, entropy,
                     top1p, argmax, bank_ptr<int>(bank, d.off_parent),
                     bank_ptr<int>(bank, d.off_depth), bank_ptr<uint32_t>(bank, d.off_mask),
                     bank_ptr<int>(bank, d.off_path), d.T, d.D, draft_tokens, accept_len, path,
                     path_capacity, bonus, best_top1p, mirror, seq);
  return launch_status("finalize_accept launch");
}

}  // namespace entmtp

extern "C" int32_t entmtp_accept(const entmtp_bank* bank, int32_t topo,
                                 const int32_t* draft_tokens, const int32_t* argmax,
                                 const float* top1p, int32_t* accept_len, int32_t* path,
                                 int32_t* bonus, float* best_top1p, void* stream) {
  clear_error();
  if (int32_t rc = check_device_bank(bank, topo)) return rc;
  ENTMTP_CHECK_ARG(draft_tokens && argmax && accept_len && path && bonus, ENTMTP_EINVAL,
                   "draft_tokens, argmax, accept_len, path and bonus must be non-NULL");
  ENTMTP_CHECK_ARG(best_top1p == nullptr || top1p != nullptr, ENTMTP_EINVAL,
                   "best_top1p needs top1p");
  return launch_accept(bank, topo, draft_tokens, argmax, top1p, accept_len, path,
                       bank->desc[topo].D + 1, bonus, best_top1p, nullptr, 0u,
                       static_cast<hipStream_t>(stream));
}

extern "C" int32_t entmtp_accept_batched(const entmtp_bank* bank, int32_t B, const int32_t* topo,
                                         const int32_t* draft_tokens, const int32_t* argmax,
                                         const float* top1p, int32_t* accept_len, int32_t* path,
                                         int32_t path_capacity, int32_t* bonus,
                                         float* best_top1p, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 1 && B <= ENTMTP_B_MAX, ENTMTP_EINVAL, "B = %d outside [1, %d]", B,
                   ENTMTP_B_MAX);
  ENTMTP_CHECK_ARG(topo != nullptr, ENTMTP_EINVAL, "topo must be a non-NULL host array");
  ENTMTP_CHECK_ARG(draft_tokens && argmax && accept_len && path && bonus, ENTMTP_EINVAL,
                   "draft_tokens, argmax, accept_len, path and bonus must be non-NULL");
  ENTMTP_CHECK_ARG(best_top1p == nullptr || top1p != nullptr, ENTMTP_EINVAL,
                   "best_top1p needs top1p");
  ENTMTP_CHECK_ARG(path_capacity >= 1 && path_capacity <= kAcceptThreads, ENTMTP_EINVAL,
                   "path_capacity = %d outside [1, %d]", path_capacity, kAcceptThreads);
  AcceptBatch a;
  int rows = 0;
  for (int b = 0; b < B; ++b) {
    if (int32_t rc = check_device_bank(bank, topo[b])) return rc;
    const TopoDesc& d = bank->desc[topo[b]];
    ENTMTP_CHECK_ARG(path_capacity >= d.D + 1, ENTMTP_EINVAL,
                     "path_capacity = %d below 1 + depth %d of sequence %d's tree", path_capacity,
                     d.D, b);
    a.s[b] = AcceptSeq{bank_ptr<int>(bank, d.off_parent), bank_ptr<int>(bank, d.off_depth),
                       bank_ptr<uint32_t>(bank, d.off_mask), bank_ptr<int>(bank, d.off_path), d.T,
                       d.D, rows};
    rows += d.T;
  }
  a.tok = draft_tokens;
  a.amax = argmax;
  a.top1p = top1p;
  a.accept_len = accept_len;
  a.path = path;
  a.path_cap = path_capacity;
  a.bonus = bonus;
  a.best = best_top1p;
  hipLaunchKernelGGL(accept_batched_kernel, dim3(B), dim3(kAcceptThreads), 0,
                     static_cast<hipStream_t>(stream), a);
  return launch_status("accept_batched launch");
}

extern "C" int32_t entmtp_accept_batched_device(const entmtp_bank* bank, int32_t B,
                                                const int32_t* topo, const int32_t* row_off,
                                                int32_t rows_cap, const int32_t* draft_tokens,
                                                const int32_t* argmax, const float* top1p,
                                                int32_t* accept_len, int32_t* path,
                                                int32_t path_capacity, int32_t* bonus,
                                                float* best_top1p, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 1 && B <= ENTMTP_B_MAX, ENTMTP_EINVAL, "B = %d outside [1, %d]", B,
                   ENTMTP_B_MAX);
  if (int32_t rc = check_device_bank(bank, 0)) return rc;
  ENTMTP_CHECK_ARG(static_cast<int>(bank->desc.size()) <= kMaxTreesAccept, ENTMTP_ERANGE,
                   "a device-planned batch names at most %d bank trees (bank has %zu)",
                   kMaxTreesAccept, bank->desc.size());
  ENTMTP_CHECK_ARG(topo && row_off, ENTMTP_EINVAL, "topo and row_off must be non-NULL device arrays");
  ENTMTP_CHECK_ARG(rows_cap >= 1, ENTMTP_EINVAL, "rows_cap = %d < 1", rows_cap);
  ENTMTP_CHECK_ARG(draft_tokens && argmax && accept_len && path && bonus, ENTMTP_EINVAL,
                   "draft_tokens, argmax, accept_len, path and bonus must be non-NULL");
  ENTMTP_CHECK_ARG(best_top1p == nullptr || top1p != nullptr, ENTMTP_EINVAL,
                   "best_top1p needs top1p");
  ENTMTP_CHECK_ARG(path_capacity >= 1 && path_capacity <= kAcceptThreads, ENTMTP_EINVAL,
                   "path_capacity = %d outside [1, %d]", path_capacity, kAcceptThreads);
  AcceptBatchDev a;
  a.n_trees = static_cast<int>(bank->desc.size());
  for (int k = 0; k < a.n_trees; ++k) {
    const TopoDesc& d = bank->desc[k];
    a.trees[k] = AcceptSeq{bank_ptr<int>(bank, d.off_parent), bank_ptr<int>(bank, d.off_depth),
                           bank_ptr<uint32_t>(bank, d.off_mask), bank_ptr<int>(bank, d.off_path),
                           d.T, d.D, 0};
  }
  a.topo = topo;
  a.row_off = row_off;
  a.rows_cap = rows_cap;
  a.tok = draft_tokens;
  a.amax = argmax;
  a.top1p = top1p;
  a.accept_len = accept_len;
  a.path = path;
  a.path_cap = path_capacity;
  a.bonus = bonus;
  a.best = best_top1p;
  hipLaunchKernelGGL(accept_batched_device_kernel, dim3(B), dim3(kAcceptThreads), 0,
                     static_cast<hipStream_t>(stream), a);
  return launch_status("accept_batched (device arrays) launch");
}

extern "C" int32_t entmtp_draft_logits(const entmtp_bank* bank, int32_t topo,
                                       const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                       int32_t hid, int32_t V, const int32_t* draft_tokens,
                                       const int32_t* argmax, float* z_draft, float* z_top,
                                       void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(hidden && w_lm && draft_tokens && argmax && z_draft && z_top, ENTMTP_EINVAL,
                   "pointers must be non-NULL");
  ENTMTP_CHECK_ARG(hid >= 8 && hid % 8 == 0 && V >= 1, ENTMTP_EINVAL,
                   "hid = %d (a positive multiple of 8), V = %d", hid, V);
  ENTMTP_CHECK_ARG(aligned16(hidden) && aligned16(w_lm), ENTMTP_EINVAL,
                   "hidden and w_lm must be 16-byte aligned");
  if (int32_t rc = check_device_bank(bank, topo)) return rc;
  const TopoDesc& d = bank->desc[topo];
  hipLaunchKernelGGL(draft_logits_kernel, dim3(d.T), dim3(64), 0, static_cast<hipStream_t>(stream),
                     bank_ptr<int>(bank, d.off_parent), reinterpret_cast<const uint16_t*>(hidden),
                     reinterpret_cast<const uint16_t*>(w_lm), hid, V, draft_tokens, argmax, z_draft,
                     z_top);
  return launch_status("draft_logits launch");
}

extern "C" int32_t entmtp_accept_typical(const entmtp_bank* bank, int32_t topo,
                                         const int32_t* draft_tokens, const int32_t* argmax,
                                         const float* z_draft, const float* z_top,
                                         const float* entropy, const float* top1p,
                                         float inv_temp, float eps, float alpha,
                                         int32_t* accept_len, int32_t* path, int32_t* bonus,
                                         float* best_top1p, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(draft_tokens && argmax && z_draft && z_top && entropy && top1p && accept_len &&
                       path && bonus,
                   ENTMTP_EINVAL, "inputs and outputs (except best_top1p) must be non-NULL");
  ENTMTP_CHECK_ARG(inv_temp > 0.f && inv_temp < INFINITY, ENTMTP_EINVAL,
                   "inv_temp must be positive and finite");
  ENTMTP_CHECK_ARG(eps >= 0.f && alpha >= 0.f && eps < INFINITY && alpha < INFINITY, ENTMTP_EINVAL,
                   "eps and alpha must be finite and >= 0");
  if (int32_t rc = check_device_bank(bank, topo)) return rc;
  const TopoDesc& d = bank->desc[topo];
  hipLaunchKernelGGL(accept_typical_kernel, dim3(1), dim3(kAcceptThreads), 0,
                     static_cast<hipStream_t>(stream), bank_ptr<int>(bank, d.off_parent),
                     bank_ptr<int>(bank, d.off_depth), bank_ptr<uint32_t>(bank, d.off_mask),
                     bank_ptr<int>(bank, d.off_path), d.T, d.D, draft_tokens, argmax, z_draft, z_top,
                     entropy, top1p, inv_temp, eps, alpha, accept_len, path, bonus, best_top1p);
  return launch_status("accept_typical launch");
}
