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

// One wavefront merges the G partials of each of R rows (rows[r] NULL: no
// row) in two steps: the row maximum and its lowest index first, then Z and S
// rebased to that maximum -- one exponential per partial.  Lane l takes
// partials l, l + 64, l + 128, ... in that order and a butterfly combines the
// lanes, so the result does not depend on R or on the path below; every
// kernel that finishes statistics merges this way and they agree bit for
// bit.  Up to 512 partials per row the loads of all R rows are issued at
// once and kept in registers (one round trip); longer rows are read twice.
constexpr int kMergeRegParts = 8;   // partials per lane held in registers

template <int R>
__device__ __forceinline__ void merge_rows(const StatPart* const (&rows)[R], int G, float inv_temp,
                                           StatPart (&out)[R]) {
  const int lane = threadIdx.x & 63;
  const StatPart kEmpty{-INFINITY, 0.f, 0.f, 0x7fffffff};
  float m[R];
  int mi[R];
  float Z[R], S[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    m[r] = -INFINITY;
    mi[r] = 0x7fffffff;
    Z[r] = 0.f;
    S[r] = 0.f;
  }
  // d <= 0; the hardware exponential (a few ulp) is far inside the 1e-3 bar
  // of the statistics
  auto add = [&](const StatPart& p, float my, float& z, float& sacc) {
    if (p.zmax != -INFINITY) {
      const float d = p.zmax * inv_temp - my;
      const float f = __expf(d);
      z += p.Z * f;
      sacc += f * (p.S + d * p.Z);
    }
  };
  auto max_butterfly = [&]() {
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1)
        take_max(m[r], mi[r], __shfl_xor(m[r], off, 64), __shfl_xor(mi[r], off, 64));
  };
  if (G <= 64 * kMergeRegParts) {
    StatPart v[R][kMergeRegParts];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int k = 0; k < kMergeRegParts; ++k) {
        const int g = lane + 64 * k;
        v[r][k] = (rows[r] && g < G) ? rows[r][g] : kEmpty;
      }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int k = 0; k < kMergeRegParts; ++k) take_max(m[r], mi[r], v[r][k].zmax, v[r][k].idx);
    max_butterfly();
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (m[r] != -INFINITY) {
        const float my = m[r] * inv_temp;
#pragma unroll
        for (int k = 0; k < kMergeRegParts; ++k) add(v[r][k], my, Z[r], S[r]);
      }
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (rows[r])
        for (int g = lane; g < G; g += 64) take_max(m[r], mi[r], rows[r][g].zmax, rows[r][g].idx);
    max_butterfly();
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (rows[r] && m[r] != -INFINITY) {
        const float my = m[r] * inv_temp;
        for (int g = lane; g < G; g += 64) add(rows[r][g], my, Z[r], S[r]);
      }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      Z[r] += __shfl_xor(Z[r], off, 64);
      S[r] += __shfl_xor(S[r], off, 64);
    }
    out[r] = StatPart{m[r], Z[r], S[r], mi[r]};
  }
}

// Two rows (b_row may be NULL), as merge_rows.
__device__ __forceinline__ void merge_rows_wave(const StatPart* __restrict__ a_row,
                                                const StatPart* __restrict__ b_row, int G,
                                                float inv_temp, StatPart& a, StatPart& b) {
  const StatPart* rows[2] = {a_row, b_row};
  StatPart o[2];
  merge_rows<2>(rows, G, inv_temp, o);
  a = o[0];
  b = o[1];
}

// A merged row's statistics: entropy ln Z - S / Z and top-1 probability 1 / Z.
__device__ __forceinline__ float part_entropy(const StatPart& p) { return logf(p.Z) - p.S / p.Z; }
__device__ __forceinline__ float part_top1p(const StatPart& p) { return 1.f / p.Z; }

// The statistics of nodes 0..T-1 by one workgroup of NTH threads, one
// wavefront per node (four nodes per pass), written to the outputs (each may
// be NULL) and, for the workgroup's own later use, to LDS arrays s_top1p and
// s_argmax (may be NULL).  The caller synchronises the workgroup before
// reading the LDS arrays.
template <int NTH>
__device__ __forceinline__ void finalize_nodes(const StatPart* __restrict__ part, int G, int T,
                                               float inv_temp, float* __restrict__ entropy,
                                               float* __restrict__ top1p, int* __restrict__ argmax,
                                               float* s_top1p, int* s_argmax) {
  constexpr int NW = NTH / 64;
  // rows per wavefront per pass (their loads go out together); one in a
  // 1024-thread workgroup, whose lanes have 128 registers
  constexpr int R = NTH >= 1024 ? 1 : 4;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int n0 = w; n0 < T; n0 += R * NW) {
    const StatPart* rows[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int n = n0 + r * NW;
      rows[r] = n < T ? part + static_cast<size_t>(n) * G : nullptr;
    }
    StatPart o[R];
    merge_rows<R>(rows, G, inv_temp, o);
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int n = n0 + r * NW;
        if (n >= T) break;
        if (entropy) entropy[n] = part_entropy(o[r]);
        if (top1p) top1p[n] = part_top1p(o[r]);
        if (argmax) argmax[n] = o[r].idx;
        if (s_top1p) s_top1p[n] = part_top1p(o[r]);
        if (s_argmax) s_argmax[n] = o[r].idx;
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
