// KV-cache update of the accepted path (the KV-cache update step of the
// proposal -> tree decoding -> verification -> update loop, §3.2).
//
// After verification the cache holds the prefix followed by the whole tree
// (slots prefix_len .. prefix_len + T - 1).  Only the accepted root-to-node
// path survives: slot prefix_len + j takes the row of slot
// prefix_len + path[j].  A source slot can be another row's destination, so
// each workgroup -- one (layer, KV head) -- reads every moved row into
// registers before writing any.  The accept length is read on the device, so
// the host does not wait for the verification result.
#include "common.hpp"

namespace entmtp {
namespace {

constexpr int kCompactThreads = 256;
constexpr int kCompactItems = 8;  // 16-byte items per thread: covers 2 * 32 rows * 256 dims

__global__ __launch_bounds__(kCompactThreads) void kv_compact_kernel(
    const int* __restrict__ path, int path_cap, const int* __restrict__ accept_len, int L,
    uint16_t* __restrict__ kc, uint16_t* __restrict__ vc, long long layer_stride, int Hkv,
    int cap, int d) {
  const int layer = blockIdx.x / Hkv, g = blockIdx.x % Hkv;
  const size_t base = static_cast<size_t>(layer) * layer_stride + static_cast<size_t>(g) * cap * d;
  int a = *accept_len;
  const int a_max = (path_cap < ENTMTP_D_MAX + 1 ? path_cap : ENTMTP_D_MAX + 1) - 1;
  a = a < 0 ? 0 : (a > a_max ? a_max : a);
  const int chunks = d >> 3;  // 16-byte chunks per row
  const int per_tensor = (a + 1) * chunks;
  const int n_items = 2 * per_tensor;

  u32x4 val[kCompactItems];
  uint16_t* dst[kCompactItems];
#pragma unroll
  for (int q = 0; q < kCompactItems; ++q) {
    const int it = threadIdx.x + q * kCompactThreads;
    dst[q] = nullptr;
    if (it < n_items) {
      const int tsel = it / per_tensor, rem = it % per_tensor;
      const int j = rem / chunks, ch = rem % chunks;
      const int src_row = L + path[j], dst_row = L + j;
      if (src_row != dst_row && path[j] >= 0 && src_row < cap && dst_row < cap) {
        uint16_t* buf = (tsel ? vc : kc) + base + ch * 8;
        val[q] = *reinterpret_cast<const u32x4*>(buf + static_cast<size_t>(src_row) * d);
        dst[q] = buf + static_cast<size_t>(dst_row) * d;
      }
    }
  }
  __syncthreads();  // every read of this (layer, head) precedes every write
#pragma unroll
  for (int q = 0; q < kCompactItems; ++q)
    if (dst[q]) *reinterpret_cast<u32x4*>(dst[q]) = val[q];
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

extern "C" int32_t entmtp_kv_compact(const int32_t* path, int32_t path_capacity,
                                     const int32_t* accept_len, int32_t prefix_len, entmtp_bf16* k_cache,
                                     entmtp_bf16* v_cache, int32_t n_layers,
                                     int64_t layer_stride, int32_t Hkv, int32_t cap, int32_t d,
                                     void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(path && accept_len && k_cache && v_cache, ENTMTP_EINVAL,
                   "path, accept_len and caches must be non-NULL");
  ENTMTP_CHECK_ARG(path_capacity >= 1, ENTMTP_EINVAL, "path_capacity = %d < 1", path_capacity);
  ENTMTP_CHECK_ARG(n_layers >= 1 && Hkv >= 1 && cap >= 1 && prefix_len >= 0, ENTMTP_EINVAL,
                   "bad sizes (n_layers %d, Hkv %d, cap %d, prefix_len %d)", n_layers, Hkv,
                   cap, prefix_len);
  ENTMTP_CHECK_ARG(d >= 8 && d % 8 == 0 && d <= 256, ENTMTP_EINVAL,
                   "d = %d must be a multiple of 8 in [8, 256]", d);
  ENTMTP_CHECK_ARG(n_layers == 1 || layer_stride >= static_cast<int64_t>(Hkv) * cap * d,
                   ENTMTP_EINVAL, "layer_stride %lld smaller than one layer",
                   static_cast<long long>(layer_stride));
  ENTMTP_CHECK_ARG(aligned16(k_cache) && aligned16(v_cache) && layer_stride % 8 == 0,
                   ENTMTP_EINVAL, "caches and layer_stride must keep 16-byte alignment");
  static_assert(2 * (ENTMTP_D_MAX + 1) * (256 / 8) <= kCompactThreads * kCompactItems,
                "compaction staging too small");
  hipLaunchKernelGGL(kv_compact_kernel, dim3(n_layers * Hkv), dim3(kCompactThreads), 0,
                     static_cast<hipStream_t>(stream), path, path_capacity, accept_len, prefix_len, k_cache,
                     v_cache, static_cast<long long>(layer_stride), Hkv, cap, d);
  return launch_status("kv_compact launch");
}
