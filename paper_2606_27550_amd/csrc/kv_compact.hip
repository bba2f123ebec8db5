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
constexpr int kCompactItems = 8;  // 16-byte items per thread at most: 2 * 32 rows * 256 dims

// Sequences of one call: their caches and prefix lengths; the paths and
// accept lengths are device arrays, one row / entry per sequence.
struct CompactArgs {
  uint16_t* kc[ENTMTP_B_MAX];
  uint16_t* vc[ENTMTP_B_MAX];
  int L[ENTMTP_B_MAX];
  const int* path;       // [B][path_cap]
  const int* accept_len; // [B]
  const DevStep* dev;    // when set, sequence 0's prefix length is dev->L
  const int* L_dev;      // when set, sequence b's prefix length is L_dev[b] (device)
  long long layer_stride;
  int path_cap, n_layers, Hkv, cap, d;
  int by_value;          // 1: one sequence whose path and accept length are below
  int a_v;
  int path_v[ENTMTP_D_MAX + 1];
};

__global__ __launch_bounds__(kCompactThreads) void kv_compact_kernel(CompactArgs p) {
  // workgroup -> (sequence, layer, KV head)
  const int per_seq = p.n_layers * p.Hkv;
  const int b = blockIdx.x / per_seq, rest = blockIdx.x % per_seq;
  const int layer = rest / p.Hkv, g = rest % p.Hkv;
  const int d = p.d, cap = p.cap, L = p.dev ? p.dev->L : (p.L_dev ? p.L_dev[b] : p.L[b]);
  // a device-held prefix length the host could not check: outside [0, cap)
  // no row can move (and L + j stays far from overflow below cap)
  if (L < 0 || L >= cap) return;
  const int* path = p.path + static_cast<size_t>(b) * p.path_cap;
  const size_t base = static_cast<size_t>(layer) * p.layer_stride + static_cast<size_t>(g) * cap * d;
  int a = p.by_value ? p.a_v : p.accept_len[b];
  const int a_max = (p.path_cap < ENTMTP_D_MAX + 1 ? p.path_cap : ENTMTP_D_MAX + 1) - 1;
  a = a < 0 ? 0 : (a > a_max ? a_max : a);
  const int chunks = d >> 3;  // 16-byte chunks per row
  const int per_tensor = (a + 1) * chunks;
  const int n_items = 2 * per_tensor;

  // the path into LDS once (one entry per thread), then the moved rows
  // staged through LDS: every read of this (sequence, layer, head) precedes
  // every write, and the kernel holds few registers, so it fits on a CU
  // beside a running LM-head workgroup
  __shared__ int s_path[ENTMTP_D_MAX + 1];
  extern __shared__ u32x4 s_val[];   // n_items entries, sized at launch
  const int t = threadIdx.x;
  if (t <= a) s_path[t] = p.by_value ? p.path_v[t] : path[t];
  __syncthreads();
  for (int it = t; it < n_items; it += kCompactThreads) {
    const int tsel = it / per_tensor, rem = it % per_tensor;
    const int j = rem / chunks, ch = rem % chunks;
    const int src_row = L + s_path[j];
    if (s_path[j] >= 0 && src_row < cap) {
      const uint16_t* buf = (tsel ? p.vc[b] : p.kc[b]) + base + ch * 8;
      s_val[it] = *reinterpret_cast<const u32x4*>(buf + static_cast<size_t>(src_row) * d);
    }
  }
  __syncthreads();
  for (int it = t; it < n_items; it += kCompactThreads) {
    const int tsel = it / per_tensor, rem = it % per_tensor;
    const int j = rem / chunks, ch = rem % chunks;
    const int src_row = L + s_path[j], dst_row = L + j;
    if (src_row != dst_row && s_path[j] >= 0 && src_row < cap && dst_row < cap) {
      uint16_t* buf = (tsel ? p.vc[b] : p.kc[b]) + base + ch * 8;
      *reinterpret_cast<u32x4*>(buf + static_cast<size_t>(dst_row) * d) = s_val[it];
    }
  }
}

int32_t check_shape(int32_t path_capacity, int32_t n_layers, int64_t layer_stride, int32_t Hkv,
                    int32_t cap, int32_t d) {
  ENTMTP_CHECK_ARG(path_capacity >= 1, ENTMTP_EINVAL, "path_capacity = %d < 1", path_capacity);
  ENTMTP_CHECK_ARG(n_layers >= 1 && Hkv >= 1 && cap >= 1, ENTMTP_EINVAL,
                   "bad sizes (n_layers %d, Hkv %d, cap %d)", n_layers, Hkv, cap);
  ENTMTP_CHECK_ARG(d >= 8 && d % 8 == 0 && d <= 256, ENTMTP_EINVAL,
                   "d = %d must be a multiple of 8 in [8, 256]", d);
  ENTMTP_CHECK_ARG(n_layers == 1 || layer_stride >= static_cast<int64_t>(Hkv) * cap * d,
                   ENTMTP_EINVAL, "layer_stride %lld smaller than one layer",
                   static_cast<long long>(layer_stride));
  ENTMTP_CHECK_ARG(layer_stride % 8 == 0, ENTMTP_EINVAL, "layer_stride must keep 16-byte alignment");
  static_assert(2 * (ENTMTP_D_MAX + 1) * (256 / 8) <= kCompactThreads * kCompactItems,
                "compaction staging too small");
  return ENTMTP_OK;
}

int32_t launch_compact(const CompactArgs& a, int B, hipStream_t s) {
  // LDS for the most rows the kernel can move: the accept length given by
  // value, else the path capacity (both clamped as in the kernel)
  const int cap_rows = a.path_cap < ENTMTP_D_MAX + 1 ? a.path_cap : ENTMTP_D_MAX + 1;
  int rows = a.by_value ? a.a_v + 1 : cap_rows;
  rows = rows < 1 ? 1 : (rows > cap_rows ? cap_rows : rows);
  const size_t lds = static_cast<size_t>(2) * rows * (a.d / 8) * sizeof(u32x4);
  hipLaunchKernelGGL(kv_compact_kernel, dim3(B * a.n_layers * a.Hkv), dim3(kCompactThreads), lds, s, a);
  return launch_status("kv_compact launch");
}

}  // namespace

int32_t launch_compact_device(const DevStep* dev, const int32_t* path, int32_t path_capacity,
                              const int32_t* accept_len, entmtp_bf16* k_cache,
                              entmtp_bf16* v_cache, int32_t n_layers, int64_t layer_stride,
                              int32_t Hkv, int32_t cap, int32_t d, hipStream_t s) {
  CompactArgs a{};
  a.kc[0] = k_cache;
  a.vc[0] = v_cache;
  a.path = path;
  a.accept_len = accept_len;
  a.dev = dev;
  a.layer_stride = static_cast<long long>(layer_stride);
  a.path_cap = path_capacity;
  a.n_layers = n_layers;
  a.Hkv = Hkv;
  a.cap = cap;
  a.d = d;
  return launch_compact(a, 1, s);
}

int32_t launch_compact_host(const int32_t* path_host, int32_t accept_len, int32_t prefix_len,
                            entmtp_bf16* k_cache, entmtp_bf16* v_cache, int32_t n_layers,
                            int64_t layer_stride, int32_t Hkv, int32_t cap, int32_t d,
                            hipStream_t s) {
  CompactArgs a{};
  a.kc[0] = k_cache;
  a.vc[0] = v_cache;
  a.L[0] = prefix_len;
  a.by_value = 1;
  a.a_v = accept_len;
  for (int j = 0; j <= ENTMTP_D_MAX; ++j) a.path_v[j] = j <= accept_len ? path_host[j] : -1;
  a.layer_stride = static_cast<long long>(layer_stride);
  a.path_cap = ENTMTP_D_MAX + 1;
  a.n_layers = n_layers;
  a.Hkv = Hkv;
  a.cap = cap;
  a.d = d;
  return launch_compact(a, 1, s);
}

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
  ENTMTP_CHECK_ARG(prefix_len >= 0, ENTMTP_EINVAL, "prefix_len = %d < 0", prefix_len);
  if (int32_t rc = check_shape(path_capacity, n_layers, layer_stride, Hkv, cap, d)) return rc;
  ENTMTP_CHECK_ARG(aligned16(k_cache) && aligned16(v_cache), ENTMTP_EINVAL,
                   "caches must be 16-byte aligned");
  CompactArgs a{};
  a.kc[0] = k_cache;
  a.vc[0] = v_cache;
  a.L[0] = prefix_len;
  a.path = path;
  a.accept_len = accept_len;
  a.layer_stride = static_cast<long long>(layer_stride);
  a.path_cap = path_capacity;
  a.n_layers = n_layers;
  a.Hkv = Hkv;
  a.cap = cap;
  a.d = d;
  return launch_compact(a, 1, static_cast<hipStream_t>(stream));
}

extern "C" int32_t entmtp_kv_compact_batched(int32_t B, const int32_t* path, int32_t path_capacity,
                                             const int32_t* accept_len, const int32_t* prefix_len,
                                             entmtp_bf16* const* k_caches,
                                             entmtp_bf16* const* v_caches, int32_t n_layers,
                                             int64_t layer_stride, int32_t Hkv, int32_t cap,
                                             int32_t d, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 1 && B <= ENTMTP_B_MAX, ENTMTP_EINVAL, "B = %d outside [1, %d]", B,
                   ENTMTP_B_MAX);
  ENTMTP_CHECK_ARG(path && accept_len, ENTMTP_EINVAL, "path and accept_len must be non-NULL");
  ENTMTP_CHECK_ARG(prefix_len && k_caches && v_caches, ENTMTP_EINVAL,
                   "prefix_len, k_caches and v_caches must be non-NULL host arrays");
  if (int32_t rc = check_shape(path_capacity, n_layers, layer_stride, Hkv, cap, d)) return rc;
  CompactArgs a{};
  for (int b = 0; b < B; ++b) {
    ENTMTP_CHECK_ARG(prefix_len[b] >= 0, ENTMTP_EINVAL, "sequence %d: prefix_len = %d < 0", b,
                     prefix_len[b]);
    ENTMTP_CHECK_ARG(k_caches[b] && v_caches[b] && aligned16(k_caches[b]) && aligned16(v_caches[b]),
                     ENTMTP_EINVAL, "sequence %d: caches must be non-NULL and 16-byte aligned", b);
    a.kc[b] = k_caches[b];
    a.vc[b] = v_caches[b];
    a.L[b] = prefix_len[b];
  }
  a.path = path;
  a.accept_len = accept_len;
  a.layer_stride = static_cast<long long>(layer_stride);
  a.path_cap = path_capacity;
  a.n_layers = n_layers;
  a.Hkv = Hkv;
  a.cap = cap;
  a.d = d;
  return launch_compact(a, B, static_cast<hipStream_t>(stream));
}

extern "C" int32_t entmtp_kv_compact_batched_device(int32_t B, const int32_t* path,
                                                    int32_t path_capacity,
                                                    const int32_t* accept_len,
                                                    const int32_t* prefix_len,
                                                    entmtp_bf16* const* k_caches,
                                                    entmtp_bf16* const* v_caches,
                                                    int32_t n_layers, int64_t layer_stride,
                                                    int32_t Hkv, int32_t cap, int32_t d,
                                                    void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 1 && B <= ENTMTP_B_MAX, ENTMTP_EINVAL, "B = %d outside [1, %d]", B,
                   ENTMTP_B_MAX);
  ENTMTP_CHECK_ARG(path && accept_len && prefix_len, ENTMTP_EINVAL,
                   "path, accept_len and prefix_len must be non-NULL device arrays");
  ENTMTP_CHECK_ARG(k_caches && v_caches, ENTMTP_EINVAL,
                   "k_caches and v_caches must be non-NULL host arrays");
  if (int32_t rc = check_shape(path_capacity, n_layers, layer_stride, Hkv, cap, d)) return rc;
  CompactArgs a{};
  for (int b = 0; b < B; ++b) {
    ENTMTP_CHECK_ARG(k_caches[b] && v_caches[b] && aligned16(k_caches[b]) && aligned16(v_caches[b]),
                     ENTMTP_EINVAL, "sequence %d: caches must be non-NULL and 16-byte aligned", b);
    a.kc[b] = k_caches[b];
    a.vc[b] = v_caches[b];
  }
  a.L_dev = prefix_len;
  a.path = path;
  a.accept_len = accept_len;
  a.layer_stride = static_cast<long long>(layer_stride);
  a.path_cap = path_capacity;
  a.n_layers = n_layers;
  a.Hkv = Hkv;
  a.cap = cap;
  a.d = d;
  return launch_compact(a, B, static_cast<hipStream_t>(stream));
}
