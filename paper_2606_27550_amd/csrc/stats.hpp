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

// One wavefront merges the G partials of each of R rows of part (row[r] < 0:
// no row; row[0] is a row) in two steps: the row maximum and its lowest index first, then Z and S
// rebased to that maximum -- one exponential per partial.  Lane l takes
// partials l, l + 64, l + 128, ... in that order and a butterfly combines the
// lanes, so the result does not depend on R or on the path below; every
// kernel that finishes statistics merges this way and they agree bit for
// bit.  Up to 64 P partials per row (512 by default) the loads of all R
// rows are issued at once and kept in registers (one round trip); longer
// rows are read twice.
constexpr int kMergeRegParts = 8;   // partials per lane held in registers

// (z, index) as one key whose unsigned order is take_max's order: larger z
// first, then the lower index (-0 is taken as +0, as take_max compares them
// equal).  The row maximum is then a max over 64-bit keys, branch-free.
__device__ __forceinline__ unsigned long long max_key(float z, int idx) {
  uint32_t u = __float_as_uint(z + 0.f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<unsigned long long>(u) << 32) | (0xffffffffu - static_cast<uint32_t>(idx));
}

__device__ __forceinline__ void key_parts(unsigned long long key, float& z, int& idx) {
  const uint32_t u = static_cast<uint32_t>(key >> 32);
  z = __uint_as_float((u & 0x80000000u) ? (u ^ 0x80000000u) : ~u);
  idx = static_cast<int>(0xffffffffu - static_cast<uint32_t>(key));
}

__device__ __forceinline__ unsigned long long key_max(unsigned long long a, unsigned long long b) {
  return a > b ? a : b;
}

template <int R, int P = kMergeRegParts>
__device__ __forceinline__ void merge_rows(const StatPart* __restrict__ part, const int (&row)[R],
                                           int G, float inv_temp, StatPart (&out)[R]) {
  const int lane = threadIdx.x & 63;
  const StatPart kEmpty{-INFINITY, 0.f, 0.f, 0x7fffffff};
  const unsigned long long kEmptyKey = max_key(-INFINITY, 0x7fffffff);
  unsigned long long key[R];
  float m[R];
  int mi[R];
  float Z[R], S[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    key[r] = kEmptyKey;
    Z[r] = 0.f;
    S[r] = 0.f;
  }
  // d <= 0; the hardware exponential (a few ulp) is far inside the 1e-3 bar
  // of the statistics.  Branch-free: an empty partial adds zeros.
  auto add = [&](const StatPart& p, float my, float& z, float& sacc) {
    const bool live = p.zmax != -INFINITY;
    const float d = live ? p.zmax * inv_temp - my : 0.f;
    const float f = live ? __expf(d) : 0.f;
    z += p.Z * f;
    sacc += f * (p.S + d * p.Z);
  };
  auto max_butterfly = [&]() {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint32_t hi = __shfl_xor(static_cast<uint32_t>(key[r] >> 32), off, 64);
        const uint32_t lo = __shfl_xor(static_cast<uint32_t>(key[r]), off, 64);
        key[r] = key_max(key[r], (static_cast<unsigned long long>(hi) << 32) | lo);
      }
#pragma unroll
    for (int r = 0; r < R; ++r) key_parts(key[r], m[r], mi[r]);
  };
  if (G <= 64 * P) {
    // unconditional loads addressed from the kernel's own pointer (clamped
    // to an existing row and partial), so the compiler issues them back to
    // back as global loads; entries past the row read as empty
    StatPart v[R][P];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const StatPart* src = part + static_cast<size_t>(row[r] >= 0 ? row[r] : row[0]) * G;
#pragma unroll
      for (int k = 0; k < P; ++k) {
        const int g = lane + 64 * k;
        v[r][k] = src[g < G ? g : 0];
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int k = 0; k < P; ++k)
        if (row[r] < 0 || lane + 64 * k >= G) v[r][k] = kEmpty;
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int k = 0; k < P; ++k) key[r] = key_max(key[r], max_key(v[r][k].zmax, v[r][k].idx));
    max_butterfly();
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (m[r] != -INFINITY) {
        const float my = m[r] * inv_temp;
#pragma unroll
        for (int k = 0; k < P; ++k) add(v[r][k], my, Z[r], S[r]);
      }
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (row[r] >= 0) {
        const StatPart* src = part + static_cast<size_t>(row[r]) * G;
        for (int g = lane; g < G; g += 64) key[r] = key_max(key[r], max_key(src[g].zmax, src[g].idx));
      }
    max_butterfly();
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (row[r] >= 0 && m[r] != -INFINITY) {
        const StatPart* src = part + static_cast<size_t>(row[r]) * G;
        const float my = m[r] * inv_temp;
        for (int g = lane; g < G; g += 64) add(src[g], my, Z[r], S[r]);
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

// Rows a and b of part (b < 0: none), as merge_rows.
__device__ __forceinline__ void merge_rows_wave(const StatPart* __restrict__ part, int a_row,
                                                int b_row, int G, float inv_temp, StatPart& a,
                                                StatPart& b) {
  const int rows[2] = {a_row, b_row};
  StatPart o[2];
  merge_rows<2>(part, rows, G, inv_temp, o);
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
template <int NTH, int R, int P>
__device__ __forceinline__ void finalize_rows(const StatPart* __restrict__ part, int G, int T,
                                              float inv_temp, float* __restrict__ entropy,
                                              float* __restrict__ top1p, int* __restrict__ argmax,
                                              float* s_top1p, int* s_argmax) {
  constexpr int NW = NTH / 64;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int n0 = w; n0 < T; n0 += R * NW) {
    int rows[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int n = n0 + r * NW;
      rows[r] = n < T ? n : -1;
    }
    StatPart o[R];
    merge_rows<R, P>(part, rows, G, inv_temp, o);
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

template <int NTH>
__device__ __forceinline__ void finalize_nodes(const StatPart* __restrict__ part, int G, int T,
                                               float inv_temp, float* __restrict__ entropy,
                                               float* __restrict__ top1p, int* __restrict__ argmax,
                                               float* s_top1p, int* s_argmax) {
  // rows per wavefront per pass (their loads go out together): one in a
  // 1024-thread workgroup, whose lanes have 128 registers; else four rows of
  // up to 512 partials, or eight rows of up to 256 (the step's small-tree LM
  // head folds two slices per partial), 128 registers of partials either way
  if constexpr (NTH >= 1024) {
    if (G <= 64 * 4)
      finalize_rows<NTH, 1, 4>(part, G, T, inv_temp, entropy, top1p, argmax, s_top1p, s_argmax);
    else
      finalize_rows<NTH, 1, kMergeRegParts>(part, G, T, inv_temp, entropy, top1p, argmax, s_top1p,
                                            s_argmax);
  } else {
    if (G <= 64 * 4)
      finalize_rows<NTH, 8, 4>(part, G, T, inv_temp, entropy, top1p, argmax, s_top1p, s_argmax);
    else
      finalize_rows<NTH, 4, kMergeRegParts>(part, G, T, inv_temp, entropy, top1p, argmax, s_top1p,
                                            s_argmax);
  }
}

// The statistics of nodes 0..T-1 from the LM head's partials, one wavefront
// per node (as entmtp_stats_finalize, arguments unchecked).
int32_t launch_stats_finalize(const void* partials, int T, int V, float inv_temp, float* entropy,
                              float* top1p, int* argmax, hipStream_t s);

// Partials per row the streaming LM head writes for vocabulary size V on the
// current device (its grid width).
int stats_slices(int V);

// Trees of up to kStepSmallT nodes: the step's LM head runs one workgroup per
// two vocabulary slices and writes one partial per workgroup per node,
// step_small_parts(V) per row (rows that long).
constexpr int kStepSmallT = 32;
int step_small_parts(int V);

// The LM head with statistics partials inside a verification step: as
// entmtp_verify_logits_partials (arguments checked by the step), but for trees
// of up to 32 nodes with one workgroup per CU looping over two vocabulary
// slices, which leaves room on every CU for the attention overlapping it.
// ev0 / ev1 (may be NULL) are recorded right before and after the LM head.
int32_t launch_step_partials(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, int T, int hid,
                             int V, float inv_temp, float* logits, void* partials, int* n_parts,
                             hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

// The LM head with statistics partials (as entmtp_verify_logits_partials,
// no logits) for a node count the device holds in *T_dev (1 <= T <= T_max
// <= 128, known only when the kernel runs).
int32_t launch_partials_device_T(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                 const int* T_dev, int T_max, int hid, int V, float inv_temp,
                                 void* partials, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

// The LM head over many rows as a tiled contraction (lm_head_gemm.hip): true
// when it takes T rows of hidden size hid for a streaming grid of G slices on
// a device with `cus` compute units; it then writes the streaming kernels'
// partial layout (G per row).
bool lm_gemm_takes(int T, int hid, int G, int cus);
int32_t launch_lm_gemm(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, float* logits, int T,
                       int hid, int V, int G, float inv_temp, void* partials, int cus,
                       hipStream_t s);

}  // namespace entmtp
