// Scoring step of the greedy acceptance-frontier construction (§3.1,
// Algorithm 1).
//
// The offline search grows a draft tree T one node at a time.  Every node of
// T (and the root) proposes its next-ranked child; all of these one-node
// augmentations T u {nu} are scored from a single rollout of the joint tree
// T u F: each sample is one verification of the joint tree, and since a
// candidate's ancestors all lie in T, the accept length of T u {nu} in that
// sample is the larger of T's own accept length and depth(nu) when nu is
// accepted.  The node added is the candidate with the largest mean accept
// length, ties broken by the smaller child-rank sum, then the smaller depth
// (then, here, the lower node index).
//
// Three launches: clear the sums, score the samples (one wavefront per sample
// at a time, integer sums added with atomics -- exact and order-free), choose
// the node (one workgroup).
#include "common.hpp"

namespace entmtp {
namespace {

constexpr int kFrontierThreads = ENTMTP_T_MAX;   // the choice: one thread per node
constexpr int kFrontierMaxGroups = 512;

__global__ __launch_bounds__(64) void frontier_clear_kernel(int* __restrict__ sums, int n) {
  for (int i = threadIdx.x; i < n; i += 64) sums[i] = 0;
}

// Whether node i passes the local test in sample s: the caller's flags, or
// greedily its draft token equal to the target's argmax at its parent.
__device__ __forceinline__ bool local_ok(const uint8_t* __restrict__ ok, const int* __restrict__ tok,
                                         const int* __restrict__ amax, int parent, int s, int i,
                                         int T) {
  const size_t row = static_cast<size_t>(s) * T;
  if (i == 0) return true;
  if (ok) return ok[row + i] != 0;
  return tok[row + i] == amax[row + parent];
}

// One wavefront scores one sample at a time (the four wavefronts of a
// workgroup take different samples): lane l owns nodes l, l + 64, l + 128 and
// l + 192, a ballot per 64-node chunk builds the sample's set of locally
// passing nodes in registers, and a node is accepted when its ancestor
// bitmask is a subset of that set -- no LDS and no barrier per sample.  The
// next sample's flags load while the current one is scored.
__global__ __launch_bounds__(kFrontierThreads) void frontier_score_kernel(
    const int* __restrict__ parent, const int* __restrict__ depth,
    const uint32_t* __restrict__ mask, const uint8_t* __restrict__ in_tree, int T, int S,
    const uint8_t* __restrict__ ok, const int* __restrict__ tok, const int* __restrict__ amax,
    int* __restrict__ sums) {
  constexpr int kChunks = ENTMTP_T_MAX / 64;
  static_assert(ENTMTP_MASK_WORDS == 2 * kChunks, "two mask words per 64-node chunk");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int waves = kFrontierThreads / 64;
  int par[kChunks], dep[kChunks];
  bool live[kChunks], member[kChunks];
  uint32_t m[kChunks][ENTMTP_MASK_WORDS];
  int total[kChunks];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int i = 64 * c + lane;
    live[c] = i < T;
    par[c] = live[c] ? parent[i] : 0;
    dep[c] = live[c] ? depth[i] : 0;
    member[c] = live[c] && (i == 0 || in_tree[i] != 0);
#pragma unroll
    for (int w = 0; w < ENTMTP_MASK_WORDS; ++w) m[c][w] = live[c] ? mask[i * ENTMTP_MASK_WORDS + w] : 0u;
    total[c] = 0;
  }
  auto flags = [&](int s, bool (&f)[kChunks]) {
#pragma unroll
    for (int c = 0; c < kChunks; ++c)
      f[c] = s < S && live[c] && local_ok(ok, tok, amax, par[c], s, 64 * c + lane, T);
  };
  const int stride = static_cast<int>(gridDim.x) * waves;
  int s = static_cast<int>(blockIdx.x) * waves + wave;
  bool nxt[kChunks], nxt2[kChunks];   // two samples' flags in flight
  flags(s, nxt);
  flags(s + stride, nxt2);
  for (; s < S; s += stride) {
    bool cur[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      cur[c] = nxt[c];
      nxt[c] = nxt2[c];
    }
    flags(s + 2 * stride, nxt2);
    uint32_t matched[ENTMTP_MASK_WORDS];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const unsigned long long b = __ballot(cur[c]);
      matched[2 * c] = static_cast<uint32_t>(b);
      matched[2 * c + 1] = static_cast<uint32_t>(b >> 32);
    }
    bool acc[kChunks];
    int a = 0;   // accept length of T in this sample: its deepest accepted node
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      acc[c] = live[c];
#pragma unroll
      for (int w = 0; w < ENTMTP_MASK_WORDS; ++w) acc[c] = acc[c] && ((m[c][w] & ~matched[w]) == 0u);
      if (member[c] && acc[c]) a = max(a, dep[c]);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) a = max(a, __shfl_xor(a, off, 64));
#pragma unroll
    for (int c = 0; c < kChunks; ++c)
      total[c] += member[c] ? a : max(a, acc[c] ? dep[c] : 0);
  }
  // the workgroup's four wavefronts first, then one atomic per node
  __shared__ int s_tot[kFrontierThreads / 64][ENTMTP_T_MAX];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) s_tot[wave][64 * c + lane] = total[c];
  __syncthreads();
  const int i = threadIdx.x;
  if (i < T) {
    int t = 0;
#pragma unroll
    for (int w = 0; w < kFrontierThreads / 64; ++w) t += s_tot[w][i];
    if (t) atomicAdd(&sums[i], t);
  }
}

// nu* over the candidates: the largest sum, then the smaller rank sum, then
// the smaller depth, then the lower index, as one 64-bit key per node.
__global__ __launch_bounds__(kFrontierThreads) void frontier_select_kernel(
    const int* __restrict__ parent, const int* __restrict__ depth,
    const int* __restrict__ path_tab, int D, const uint8_t* __restrict__ in_tree, int T,
    const int* __restrict__ sums, int* __restrict__ best) {
  __shared__ int s_parent[ENTMTP_T_MAX];
  __shared__ int s_rank[ENTMTP_T_MAX];
  __shared__ unsigned long long s_key[kFrontierThreads / 64];
  const int i = threadIdx.x, lane = i & 63, wave = i >> 6;
  const bool live = i < T;
  if (live) s_parent[i] = parent[i];
  __syncthreads();
  // rank among the parent's children = earlier siblings (index order)
  int rank = 0;
  if (live && i > 0)
    for (int j = 1; j < i; ++j) rank += s_parent[j] == s_parent[i];
  if (live) s_rank[i] = rank;
  __syncthreads();
  unsigned long long key = 0ull;
  if (live && i > 0 && in_tree[i] == 0) {
    const int dep = depth[i];
    int rs = 0;
    for (int k = 1; k <= dep; ++k) rs += s_rank[path_tab[i * (D + 1) + k]];
    // rank sums stay below 256 * 32 and depths below 32, so the fields never
    // overlap and a real candidate's key is never 0
    const unsigned low = (static_cast<unsigned>(8191 - rs) << 13) |
                         (static_cast<unsigned>(31 - dep) << 8) | static_cast<unsigned>(255 - i);
    key = (static_cast<unsigned long long>(static_cast<unsigned>(sums[i])) << 32) | low;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const unsigned long long o = __shfl_xor(key, off, 64);
    key = o > key ? o : key;
  }
  if (lane == 0) s_key[wave] = key;
  __syncthreads();
  if (i == 0) {
    unsigned long long k = s_key[0];
#pragma unroll
    for (int w = 1; w < kFrontierThreads / 64; ++w) k = s_key[w] > k ? s_key[w] : k;
    *best = k ? 255 - static_cast<int>(k & 255ull) : -1;
  }
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

extern "C" int32_t entmtp_frontier_score(const entmtp_bank* bank, int32_t topo,
                                         const uint8_t* in_tree, int32_t n_samples,
                                         const uint8_t* local_ok, const int32_t* draft_tokens,
                                         const int32_t* argmax, int32_t* sums, int32_t* best,
                                         void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(in_tree && sums && best, ENTMTP_EINVAL, "in_tree, sums and best must be non-NULL");
  ENTMTP_CHECK_ARG(n_samples >= 1, ENTMTP_EINVAL, "n_samples = %d < 1", n_samples);
  ENTMTP_CHECK_ARG(local_ok || (draft_tokens && argmax), ENTMTP_EINVAL,
                   "give local_ok, or draft_tokens and argmax");
  if (int32_t rc = check_device_bank(bank, topo)) return rc;
  const TopoDesc& d = bank->desc[topo];
  ENTMTP_CHECK_ARG(static_cast<int64_t>(n_samples) * (d.D > 0 ? d.D : 1) < (int64_t{1} << 31),
                   ENTMTP_ERANGE, "n_samples %d x depth %d overflows the int32 sums", n_samples,
                   d.D);
  auto s = static_cast<hipStream_t>(stream);
  const int* parent = bank_ptr<int>(bank, d.off_parent);
  const int* depth = bank_ptr<int>(bank, d.off_depth);
  hipLaunchKernelGGL(frontier_clear_kernel, dim3(1), dim3(64), 0, s, sums, d.T);
  if (int32_t rc = launch_status("frontier_clear launch")) return rc;
  // about 16 samples per wavefront (each workgroup's sums cost one atomic per
  // node), at most kFrontierMaxGroups workgroups
  const int per_group = 16 * (kFrontierThreads / 64);
  int groups = (n_samples + per_group - 1) / per_group;
  groups = groups < kFrontierMaxGroups ? groups : kFrontierMaxGroups;
  hipLaunchKernelGGL(frontier_score_kernel, dim3(groups), dim3(kFrontierThreads), 0, s, parent,
                     depth, bank_ptr<uint32_t>(bank, d.off_mask), in_tree, d.T, n_samples, local_ok,
                     draft_tokens, argmax, sums);
  if (int32_t rc = launch_status("frontier_score launch")) return rc;
  hipLaunchKernelGGL(frontier_select_kernel, dim3(1), dim3(kFrontierThreads), 0, s, parent, depth,
                     bank_ptr<int>(bank, d.off_path), d.D, in_tree, d.T, sums, best);
  return launch_status("frontier_select launch");
}
