// Speculative-sampling verification of a draft tree (§2.1).
//
// §2.1 states the rule for one chain: a draft token t is kept with
// probability min(1, p(t) / p_hat(t)), p the target's distribution and p_hat
// the draft's, left to right; at the first rejection the rest is dropped and
// a replacement is drawn from norm(max(0, p - p_hat)).  On a tree the walk
// starts at the root with r = p there and tries the current node's children
// in index (rank) order, all drafted from the node's draft distribution q:
// child c passes when u_c * q(t_c) < r(t_c); the first that passes becomes
// the current node (r = p at it), and each one that fails replaces r by
// norm(max(0, r - q)) before the next sibling is tried.  When no child
// passes, or the node is a leaf, the bonus token is drawn from r by inverse
// CDF over the vocabulary in index order.  For a chain this is the rule
// above; the uniforms are inputs, so a run is reproducible.
//
// One workgroup of 1024 threads walks the tree.  The target's distribution at
// a node comes from its logits and the statistics the LM head already
// produced at the same temperature (argmax and top-1 probability:
// p(v) = exp((z_v - z_argmax) * inv_temp) * top1p), so a level that accepts
// costs no pass over the vocabulary; a rejection costs two (the residual's
// mass, then -- if it has any -- the residual itself into the workspace),
// and the draw one chunked scan.  The walk is sequential in its decisions,
// so the kernel is latency-bound; every pass is a coalesced stream.
#include "common.hpp"

namespace entmtp {
namespace {

constexpr int kSpecThreads = 1024;
constexpr int kSpecWaves = kSpecThreads / 64;

// Sum in a fixed order: lanes by butterfly, then the wavefronts in order.
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int w = 1; w < kSpecWaves; ++w) s += red[w];
  return s;
}

__global__ __launch_bounds__(kSpecThreads) void accept_stochastic_kernel(
    const int* __restrict__ parent, const int* __restrict__ depth,
    const int* __restrict__ path_tab, int T, int D, const int* __restrict__ tok,
    const float* __restrict__ z, const float* __restrict__ q, int V, float inv_temp,
    const int* __restrict__ amax, const float* __restrict__ top1p,
    const float* __restrict__ u_accept, const float* __restrict__ u_sample, float* __restrict__ w,
    int* __restrict__ accept_len, int* __restrict__ path_out, int path_cap,
    int* __restrict__ bonus) {
  __shared__ float red[kSpecWaves];
  __shared__ float s_scan[kSpecWaves];
  __shared__ int s_children[ENTMTP_T_MAX];
  __shared__ int s_nchild;
  __shared__ int s_pass;
  __shared__ int s_hit;
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int cur = 0;
  // each level descends one depth, so the walk ends within D + 1 levels
  for (int level = 0; level <= D; ++level) {
    if (tid == 0) {
      int n = 0;
      for (int i = cur + 1; i < T; ++i)
        if (parent[i] == cur) s_children[n++] = i;
      s_nchild = n;
    }
    __syncthreads();   // s_children and s_nchild are written
    const float* zr = z + static_cast<size_t>(cur) * V;
    const float* qr = q + static_cast<size_t>(cur) * V;
    // target distribution at cur: p(v) = exp((z_v - z_max) * inv_temp) * top1p
    const float zm = zr[amax[cur]], p1 = top1p[cur];
    // r(v) = resid ? w[v] / Zr : p(v)
    bool resid = false;
    float Zr = 1.f;
    auto r_at = [&](int v) { return resid ? w[v] / Zr : expf((zr[v] - zm) * inv_temp) * p1; };
    int next = -1;
    const int nchild = s_nchild;
    for (int j = 0; j < nchild; ++j) {
      const int c = s_children[j];
      if (tid == 0) {
        const int t = tok[c];
        const bool in_v = t >= 0 && t < V;
        const float rt = in_v ? r_at(t) : 0.f, qt = in_v ? qr[t] : 0.f;
        s_pass = qt > 0.f ? (u_accept[c] * qt < rt) : (rt > 0.f);
      }
      __syncthreads();
      if (s_pass) {
        next = c;
        break;
      }
      // residual max(0, r - q): its mass, then (if any) the values
      float part = 0.f;
      for (int v = tid; v < V; v += kSpecThreads) part += fmaxf(r_at(v) - qr[v], 0.f);
      const float mass = block_sum(part, red);
      if (mass > 0.f) {   // (with no mass left, r stays as it is)
        for (int v = tid; v < V; v += kSpecThreads) w[v] = fmaxf(r_at(v) - qr[v], 0.f);
        resid = true;
        Zr = mass;
      }
      __syncthreads();   // the residual is written before thread 0 reads it
    }
    if (next >= 0) {
      cur = next;
      __syncthreads();   // s_children is rebuilt for the next level
      continue;
    }
    // draw from r: contiguous chunks per thread, exclusive scan of their sums
    const int chunk = (V + kSpecThreads - 1) / kSpecThreads;
    const int v0 = tid * chunk, v1 = min(V, v0 + chunk);
    float cs = 0.f;
    int last = -1;   // this chunk's last token with mass
    for (int v = v0; v < v1; ++v) {
      const float rv = r_at(v);
      cs += rv;
      if (rv > 0.f) last = v;
    }
    float incl = cs;   // inclusive scan within the wavefront
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float o = __shfl_up(incl, off, 64);
      if (lane >= off) incl += o;
    }
    if (lane == 63) s_scan[wave] = incl;
    if (tid == 0) {
      s_hit = 0x7fffffff;
      s_last = -1;
    }
    __syncthreads();
    float base = 0.f, total = 0.f;
    for (int wv = 0; wv < kSpecWaves; ++wv) {
      if (wv < wave) base += s_scan[wv];
      total += s_scan[wv];
    }
    const float excl = base + incl - cs;
    const float target = u_sample[cur] * total;
    if (cs > 0.f && excl <= target && target < excl + cs) {
      float acc = excl;
      int b = v1 - 1;
      for (int v = v0; v < v1; ++v) {
        acc += r_at(v);
        if (acc > target) {
          b = v;
          break;
        }
      }
      atomicMin(&s_hit, b);   // (rounding at a chunk boundary could let two chunks claim it)
    }
    if (last >= 0) atomicMax(&s_last, last);
    __syncthreads();
    const int a = depth[cur];
    if (tid < path_cap) path_out[tid] = tid <= a ? path_tab[cur * (D + 1) + tid] : -1;
    if (tid == 0) {
      *accept_len = a;
      // past the rounded total (no chunk claims the target): the last token with mass
      *bonus = s_hit != 0x7fffffff ? s_hit : s_last;
    }
    return;
  }
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

extern "C" int32_t entmtp_accept_stochastic(const entmtp_bank* bank, int32_t topo,
                                            const int32_t* draft_tokens, const float* logits,
                                            const float* q, int32_t V, float inv_temp,
                                            const int32_t* argmax, const float* top1p,
                                            const float* u_accept, const float* u_sample,
                                            float* workspace, int32_t* accept_len,
                                            int32_t* path, int32_t* bonus, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(draft_tokens && logits && q && argmax && top1p && u_accept && u_sample &&
                       workspace && accept_len && path && bonus,
                   ENTMTP_EINVAL, "pointers must be non-NULL");
  ENTMTP_CHECK_ARG(V >= 1, ENTMTP_EINVAL, "V = %d < 1", V);
  ENTMTP_CHECK_ARG(inv_temp > 0.f && inv_temp < INFINITY, ENTMTP_EINVAL,
                   "inv_temp must be positive and finite");
  if (int32_t rc = check_device_bank(bank, topo)) return rc;
  const TopoDesc& d = bank->desc[topo];
  hipLaunchKernelGGL(accept_stochastic_kernel, dim3(1), dim3(kSpecThreads), 0,
                     static_cast<hipStream_t>(stream), bank_ptr<int>(bank, d.off_parent),
                     bank_ptr<int>(bank, d.off_depth), bank_ptr<int>(bank, d.off_path), d.T, d.D,
                     draft_tokens, logits, q, V, inv_temp, argmax, top1p, u_accept, u_sample,
                     workspace,
                     accept_len, path, d.D + 1, bonus);
  return launch_status("accept_stochastic launch");
}
