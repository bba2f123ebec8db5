// Per-node softmax statistics of the verifier logits.
//
// The scheduler of §4 reads the target's top-1 probability p0 at the
// verifier's last position; §3 / Appendix A use the entropy of the same
// distribution as the regime signal.  For every logits row the kernel
// produces the lowest-index argmax, p1 = 1/Z and the entropy
// H = ln Z - sum (y - m) e^(y - m) / Z with y = inv_temp * z, m = max y.
//
// One workgroup per row; the row is read twice (max / argmax, then the two
// sums), the second pass normally from L2.  Reductions use wave shuffles and
// a fixed-order combine of the per-wave results, so the result does not
// depend on scheduling.
#include <cfloat>
#include <climits>

#include "common.hpp"

namespace entmtp {
namespace {

constexpr int kStatsThreads = 512;
constexpr int kStatsWaves = kStatsThreads / 64;

// (value, index) pair ordered by value descending, then index ascending:
// an associative total order, so any reduction tree gives the same winner.
__device__ __forceinline__ void take_best(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

__global__ __launch_bounds__(kStatsThreads) void logit_stats_kernel(
    const float* __restrict__ logits, int V, float inv_temp, float* __restrict__ entropy,
    float* __restrict__ top1p, int* __restrict__ argmax) {
  __shared__ float s_v[kStatsWaves];
  __shared__ int s_i[kStatsWaves];
  __shared__ float s_z[kStatsWaves], s_s[kStatsWaves];

  const float* z = logits + static_cast<size_t>(blockIdx.x) * V;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const bool vec = (V & 3) == 0;

  // ---- pass 1: max and lowest index attaining it
  float best = -INFINITY;
  int bidx = INT_MAX;
  if (vec) {
    const float4* z4 = reinterpret_cast<const float4*>(z);
    for (int u = tid; u < (V >> 2); u += kStatsThreads) {
      float4 x = z4[u];
      take_best(best, bidx, x.x, 4 * u + 0);
      take_best(best, bidx, x.y, 4 * u + 1);
      take_best(best, bidx, x.z, 4 * u + 2);
      take_best(best, bidx, x.w, 4 * u + 3);
    }
  } else {
    for (int v = tid; v < V; v += kStatsThreads) take_best(best, bidx, z[v], v);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1)
    take_best(best, bidx, __shfl_xor(best, off, 64), __shfl_xor(bidx, off, 64));
  if (lane == 0) {
    s_v[wave] = best;
    s_i[wave] = bidx;
  }
  __syncthreads();
  best = s_v[0];
  bidx = s_i[0];
  for (int w = 1; w < kStatsWaves; ++w) take_best(best, bidx, s_v[w], s_i[w]);

  // ---- pass 2: Z = sum e^(y-m), S = sum (y-m) e^(y-m)
  const float m = best * inv_temp;
  float Z = 0.f, S = 0.f;
  auto add = [&](float x) {
    const float t = x * inv_temp - m;
    const float e = expf(t);
    Z += e;
    if (e > 0.f) S += t * e;  // keeps (-inf) * 0 out of the sum
  };
  if (vec) {
    const float4* z4 = reinterpret_cast<const float4*>(z);
    for (int u = tid; u < (V >> 2); u += kStatsThreads) {
      float4 x = z4[u];
      add(x.x);
      add(x.y);
      add(x.z);
      add(x.w);
    }
  } else {
    for (int v = tid; v < V; v += kStatsThreads) add(z[v]);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    Z += __shfl_xor(Z, off, 64);
    S += __shfl_xor(S, off, 64);
  }
  if (lane == 0) {
    s_z[wave] = Z;
    s_s[wave] = S;
  }
  __syncthreads();
  if (tid == 0) {
    float Zt = 0.f, St = 0.f;
    for (int w = 0; w < kStatsWaves; ++w) {
      Zt += s_z[w];
      St += s_s[w];
    }
    if (entropy) entropy[blockIdx.x] = logf(Zt) - St / Zt;
    if (top1p) top1p[blockIdx.x] = 1.f / Zt;
    if (argmax) argmax[blockIdx.x] = bidx;
  }
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

extern "C" int32_t entmtp_logit_stats(const float* logits, int32_t T, int32_t V, float inv_temp,
                                      float* entropy, float* top1p, int32_t* argmax,
                                      void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(logits != nullptr, ENTMTP_EINVAL, "logits is NULL");
  ENTMTP_CHECK_ARG(T >= 1 && V >= 1, ENTMTP_EINVAL, "T = %d, V = %d must be >= 1", T, V);
  ENTMTP_CHECK_ARG(inv_temp > 0.f && inv_temp < INFINITY, ENTMTP_EINVAL,
                   "inv_temp = %g must be positive and finite", static_cast<double>(inv_temp));
  ENTMTP_CHECK_ARG(aligned16(logits), ENTMTP_EINVAL, "logits must be 16-byte aligned");
  if (!entropy && !top1p && !argmax) return ENTMTP_OK;
  hipLaunchKernelGGL(logit_stats_kernel, dim3(T), dim3(kStatsThreads), 0,
                     static_cast<hipStream_t>(stream), logits, V, inv_temp, entropy, top1p,
                     argmax);
  return launch_status("logit_stats launch");
}
