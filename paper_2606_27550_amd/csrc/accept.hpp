// Device helpers of greedy tree acceptance shared by the kernels that accept
// a tree: the acceptance kernels and the LM-head kernel that finishes a
// small tree's step in its last workgroup.  One thread per node; see
// accept.hip for the method.
#pragma once

#include "common.hpp"

namespace entmtp {

constexpr int kAcceptThreads = ENTMTP_T_MAX;

// A thread's node of the tree (thread i holds node i): what the acceptance
// needs that does not depend on the target's statistics, so a kernel can
// fetch it before those are ready.
struct NodeIn {
  int tok, parent, depth;
  uint32_t mask[ENTMTP_MASK_WORDS];
};

__device__ __forceinline__ NodeIn accept_load(const int* __restrict__ parent,
                                              const int* __restrict__ depth,
                                              const uint32_t* __restrict__ mask,
                                              const int* __restrict__ tok, int T) {
  NodeIn n{};
  const int i = threadIdx.x;
  if (i < T) {
    n.tok = tok[i];
    n.parent = parent[i];
    n.depth = depth[i];
#pragma unroll
    for (int w = 0; w < ENTMTP_MASK_WORDS; ++w) n.mask[w] = mask[i * ENTMTP_MASK_WORDS + w];
  }
  return n;
}

// Greedy local test: node i's draft token is the target's argmax at its parent.
__device__ __forceinline__ bool greedy_ok(const NodeIn& n, const int* amax, int T) {
  const int i = threadIdx.x;
  return i < T && (i == 0 || n.tok == amax[n.parent]);
}

// The acceptance of one tree by one workgroup of NTH threads (at least
// ENTMTP_T_MAX); `ok`: this thread's node is locally acceptable (the root
// always is).  Writes the accept length, path (entries past it -1), bonus
// token and s, publishes them to `mirror` when given, and returns (in every
// thread) depth(best) * 1024 + (1023 - best).
template <int NTH = kAcceptThreads>
__device__ __forceinline__ int accept_finish(
    const NodeIn& n, bool ok, const int* __restrict__ path_tab, int T, int D,
    const int* amax, const float* top1p,
    int* __restrict__ accept_len, int* __restrict__ path_out, int path_cap,
    int* __restrict__ bonus, float* __restrict__ best_p, StepMirror* __restrict__ mirror,
    uint32_t seq) {
  static_assert(NTH >= ENTMTP_T_MAX && NTH % 64 == 0, "one thread per possible node");
  __shared__ uint32_t matched[ENTMTP_MASK_WORDS];
  __shared__ int s_key[NTH / 64];
  const int i = threadIdx.x;
  if (i < ENTMTP_MASK_WORDS) matched[i] = 0u;
  __syncthreads();
  if (i < T && ok) atomicOr(&matched[i >> 5], 1u << (i & 31));
  __syncthreads();
  // key orders accepted nodes by depth, then by lower index
  int key = -1;
  if (i < T) {
    bool acc = true;
#pragma unroll
    for (int w = 0; w < ENTMTP_MASK_WORDS; ++w) acc = acc && ((n.mask[w] & ~matched[w]) == 0u);
    if (acc) key = n.depth * 1024 + (1023 - i);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) key = max(key, __shfl_xor(key, off, 64));
  if ((i & 63) == 0) s_key[i >> 6] = key;
  __syncthreads();
  key = s_key[0];
#pragma unroll
  for (int w = 1; w < NTH / 64; ++w) key = max(key, s_key[w]);
  const int best = 1023 - (key & 1023);
  const int a = key >> 10;
  if (i < path_cap) path_out[i] = (i <= a) ? path_tab[best * (D + 1) + i] : -1;
  if (i == 0) {
    *accept_len = a;
    *bonus = amax[best];
    if (best_p) *best_p = top1p ? top1p[best] : 0.f;
  }
  if (mirror && i < kMirrorWords) {   // one tagged word per lane
    uint32_t field;
    if (i == 0) {
      field = static_cast<uint32_t>(a);
    } else if (i == 1) {
      field = static_cast<uint32_t>(amax[best]);
    } else if (i == 2) {
      field = __float_as_uint(top1p ? top1p[best] : 0.f);
    } else {
      field = 0u;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int j = (i - 3) * 4 + b;
        const uint32_t node = j <= a ? static_cast<uint32_t>(path_tab[best * (D + 1) + j]) : 0xffu;
        field |= (node & 0xffu) << (8 * b);
      }
    }
    __hip_atomic_store(reinterpret_cast<uint64_t*>(mirror) + i,
                       (static_cast<uint64_t>(seq) << 32) | field, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_SYSTEM);
  }
  return key;
}

}  // namespace entmtp
