// Per-node softmax statistics from per-slice partials (device helpers shared
// by the LM-head kernels and the kernels that finish a verification step).
//
// A partial summarises one slice of a logit row z (already in fp32):
// zmax = the slice's largest raw logit, idx = its lowest index attaining it,
// and, with y = inv_temp * z and m = inv_temp * zmax,
// Z = sum exp(y - m) and S = sum (y - m) exp(y - m).  Two partials merge by
// rescaling to the larger maximum; the merged row gives top-1 probability
// 1 / Z and entropy ln Z - S / Z (§4's p_0 and the entropy of §3).  The
// argmax is decided on the raw fp32 logits, lowest index among equals.
#pragma once

#include "common.hpp"

namespace entmtp {

struct StatPart {
  float zmax, Z, S;
  int idx;
};

__device__ __forceinline__ void take_max(float& zm, int& zi, float z2, int i2) {
  if (z2 > zm || (z2 == zm && i2 < zi)) {
    zm = z2;
    zi = i2;
  }
}

__device__ __forceinline__ void part_merge(StatPart& a, const StatPart& b, float inv_temp) {
  float zm = a.zmax;
  int zi = a.idx;
  take_max(zm, zi, b.zmax, b.idx);
  if (zm == -INFINITY) return;   // both empty
  const float my = zm * inv_temp;
  float Z = 0.f, S = 0.f;
  if (a.zmax != -INFINITY) {
    const float ma = a.zmax * inv_temp, f = expf(ma - my);
    Z += a.Z * f;
    S += f * (a.S + (ma - my) * a.Z);
  }
  if (b.zmax != -INFINITY) {
    const float mb = b.zmax * inv_temp, f = expf(mb - my);
    Z += b.Z * f;
    S += f * (b.S + (mb - my) * b.Z);
  }
  a = StatPart{zm, Z, S, zi};
}

__device__ __forceinline__ StatPart shfl_part(const StatPart& p, int off) {
  return StatPart{__shfl_xor(p.zmax, off, 64), __shfl_xor(p.Z, off, 64), __shfl_xor(p.S, off, 64),
                  __shfl_xor(p.idx, off, 64)};
}

constexpr int kFinThreads = 256;

// Merges the G partials of row blockIdx.x with kFinThreads threads in a fixed
// order (strided fold, butterfly, then the waves in index order) and writes
// the row's statistics (each output may be NULL).  Every kernel that
// finishes statistics uses this, so their results agree bit for bit.
__device__ __forceinline__ void finalize_node(const StatPart* __restrict__ part, int G,
                                              float inv_temp, float* __restrict__ entropy,
                                              float* __restrict__ top1p,
                                              int* __restrict__ argmax) {
  __shared__ StatPart wsum[kFinThreads / 64];
  const StatPart* row = part + static_cast<size_t>(blockIdx.x) * G;
  StatPart p{-INFINITY, 0.f, 0.f, 0x7fffffff};
  for (int g = threadIdx.x; g < G; g += kFinThreads) part_merge(p, row[g], inv_temp);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) part_merge(p, shfl_part(p, off), inv_temp);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = p;
  __syncthreads();
  if (threadIdx.x == 0) {
    StatPart a = wsum[0];
    for (int w = 1; w < kFinThreads / 64; ++w) part_merge(a, wsum[w], inv_temp);
    if (entropy) entropy[blockIdx.x] = logf(a.Z) - a.S / a.Z;
    if (top1p) top1p[blockIdx.x] = 1.f / a.Z;
    if (argmax) argmax[blockIdx.x] = a.idx;
  }
}

// Partials per row the streaming LM head writes for vocabulary size V on the
// current device (its grid width).
int stats_slices(int V);

// The LM head with statistics partials inside a verification step: as
// entmtp_verify_logits_partials (arguments checked by the step), but for trees
// of up to 32 nodes with one workgroup per CU looping over two vocabulary
// slices, which leaves room on every CU for the attention overlapping it.
int32_t launch_step_partials(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, int T, int hid,
                             int V, float inv_temp, float* logits, void* partials, hipStream_t s);

// The LM head with statistics partials (as entmtp_verify_logits_partials,
// no logits) for a node count the device holds in *T_dev (1 <= T <= T_max
// <= 128, known only when the kernel runs).
int32_t launch_partials_device_T(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                 const int* T_dev, int T_max, int hid, int V, float inv_temp,
                                 void* partials, hipStream_t s);

}  // namespace entmtp
