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

// Merges the G partials of one row with one wavefront in a fixed order --
// lane l folds partials l, l + 64, l + 128, ... in turn, then a butterfly
// over the 64 lanes -- so that every lane ends with the row's partial.  Every
// kernel that finishes statistics merges this way, so their results agree
// bit for bit.  Two rows at a time (b_row may be NULL): the loads of both are
// issued before either is folded.
__device__ __forceinline__ void merge_rows_wave(const StatPart* __restrict__ a_row,
                                                const StatPart* __restrict__ b_row, int G,
                                                float inv_temp, StatPart& a, StatPart& b) {
  const int lane = threadIdx.x & 63;
  a = StatPart{-INFINITY, 0.f, 0.f, 0x7fffffff};
  b = a;
  int g = lane;
  for (; g + 192 < G; g += 256) {
    StatPart ra[4], rb[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) ra[k] = a_row[g + 64 * k];
    if (b_row) {
#pragma unroll
      for (int k = 0; k < 4; ++k) rb[k] = b_row[g + 64 * k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) part_merge(a, ra[k], inv_temp);
    if (b_row) {
#pragma unroll
      for (int k = 0; k < 4; ++k) part_merge(b, rb[k], inv_temp);
    }
  }
  for (; g < G; g += 64) {
    part_merge(a, a_row[g], inv_temp);
    if (b_row) part_merge(b, b_row[g], inv_temp);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    part_merge(a, shfl_part(a, off), inv_temp);
    part_merge(b, shfl_part(b, off), inv_temp);
  }
}

// A merged row's statistics: entropy ln Z - S / Z and top-1 probability 1 / Z.
__device__ __forceinline__ float part_entropy(const StatPart& p) { return logf(p.Z) - p.S / p.Z; }
__device__ __forceinline__ float part_top1p(const StatPart& p) { return 1.f / p.Z; }

// The statistics of nodes 0..T-1 by one workgroup of NTH threads, one
// wavefront per node (two nodes per pass), written to the outputs (each may
// be NULL) and, for the workgroup's own later use, to LDS arrays s_top1p and
// s_argmax (may be NULL).  The caller synchronises the workgroup before
// reading the LDS arrays.
template <int NTH>
__device__ __forceinline__ void finalize_nodes(const StatPart* __restrict__ part, int G, int T,
                                               float inv_temp, float* __restrict__ entropy,
                                               float* __restrict__ top1p, int* __restrict__ argmax,
                                               float* s_top1p, int* s_argmax) {
  constexpr int NW = NTH / 64;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int n0 = w; n0 < T; n0 += 2 * NW) {
    const int n1 = n0 + NW;
    StatPart a, b;
    merge_rows_wave(part + static_cast<size_t>(n0) * G,
                    n1 < T ? part + static_cast<size_t>(n1) * G : nullptr, G, inv_temp, a, b);
    if (lane == 0) {
      if (entropy) entropy[n0] = part_entropy(a);
      if (top1p) top1p[n0] = part_top1p(a);
      if (argmax) argmax[n0] = a.idx;
      if (s_top1p) s_top1p[n0] = part_top1p(a);
      if (s_argmax) s_argmax[n0] = a.idx;
      if (n1 < T) {
        if (entropy) entropy[n1] = part_entropy(b);
        if (top1p) top1p[n1] = part_top1p(b);
        if (argmax) argmax[n1] = b.idx;
        if (s_top1p) s_top1p[n1] = part_top1p(b);
        if (s_argmax) s_argmax[n1] = b.idx;
      }
    }
  }
}

// The statistics of nodes 0..T-1 from the LM head's partials, one wavefront
// per node (as entmtp_stats_finalize, arguments unchecked).
int32_t launch_stats_finalize(const void* partials, int T, int V, float inv_temp, float* entropy,
                              float* top1p, int* argmax, hipStream_t s);

// Partials per row the streaming LM head writes for vocabulary size V on the
// current device (its grid width).
int stats_slices(int V);

// The LM head with statistics partials inside a verification step: as
// entmtp_verify_logits_partials (arguments checked by the step), but for trees
// of up to 32 nodes with one workgroup per CU looping over two vocabulary
// slices, which leaves room on every CU for the attention overlapping it.
// ev0 / ev1 (may be NULL) are recorded right before and after the LM head.
int32_t launch_step_partials(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, int T, int hid,
                             int V, float inv_temp, float* logits, void* partials, hipStream_t s,
                             hipEvent_t ev0, hipEvent_t ev1);

// The LM head with statistics partials (as entmtp_verify_logits_partials,
// no logits) for a node count the device holds in *T_dev (1 <= T <= T_max
// <= 128, known only when the kernel runs).
int32_t launch_partials_device_T(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                 const int* T_dev, int T_max, int hid, int V, float inv_temp,
                                 void* partials, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

}  // namespace entmtp
