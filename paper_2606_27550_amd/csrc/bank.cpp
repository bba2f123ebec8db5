// Error reporting and the TopologyBank planner.
//
// The bank holds, per draft tree, the buffers a Medusa-style verifier ships
// with each tree -- attention mask, position offsets and gather / retrieve
// indices (paper §2.3) -- precomputed once so that the scheduler of §4 can
// switch trees by index ("Cost": a pointer swap with no GPU work).  Planning
// is pure host code; the finished image goes to the device in one copy.
#include <cstdarg>
#include <cstring>

#include "common.hpp"

namespace entmtp {

static thread_local std::string g_last_error;

int32_t fail(int32_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_error() { g_last_error.clear(); }

int32_t hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ENTMTP_OK;
  return fail(ENTMTP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

int32_t check_device_bank(const entmtp_bank* bank, int32_t topo) {
  ENTMTP_CHECK_ARG(bank != nullptr, ENTMTP_EINVAL, "bank is NULL");
  ENTMTP_CHECK_ARG(bank->arena != nullptr, ENTMTP_EINVAL,
                   "bank was built without a device arena");
  ENTMTP_CHECK_ARG(topo >= 0 && topo < static_cast<int32_t>(bank->desc.size()),
                   ENTMTP_EINVAL, "topo %d outside [0, %zu)", topo, bank->desc.size());
  return ENTMTP_OK;
}

namespace {

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// Appends one tree's arrays to `img` and fills its descriptor.
void plan_tree(const int32_t* parent, int32_t T, std::vector<uint8_t>& img, TopoDesc& d) {
  std::vector<int32_t> depth(T, 0);
  for (int32_t i = 1; i < T; ++i) depth[i] = depth[parent[i]] + 1;
  int32_t D = 0;
  for (int32_t i = 0; i < T; ++i) D = depth[i] > D ? depth[i] : D;
  const int32_t W = D + 1;

  // mask row i = mask row parent(i) plus bit i (parents precede children)
  std::vector<uint32_t> mask(static_cast<size_t>(T) * ENTMTP_MASK_WORDS, 0u);
  for (int32_t i = 0; i < T; ++i) {
    uint32_t* row = &mask[static_cast<size_t>(i) * ENTMTP_MASK_WORDS];
    if (i > 0) std::memcpy(row, &mask[static_cast<size_t>(parent[i]) * ENTMTP_MASK_WORDS],
                           ENTMTP_MASK_WORDS * sizeof(uint32_t));
    row[i >> 5] |= 1u << (i & 31);
  }
  // path row i = path row parent(i) with i at depth(i)
  std::vector<int32_t> path(static_cast<size_t>(T) * W, -1);
  for (int32_t i = 0; i < T; ++i) {
    int32_t* row = &path[static_cast<size_t>(i) * W];
    if (i > 0) std::memcpy(row, &path[static_cast<size_t>(parent[i]) * W], W * sizeof(int32_t));
    row[depth[i]] = i;
  }
  std::vector<char> has_child(T, 0);
  for (int32_t i = 1; i < T; ++i) has_child[parent[i]] = 1;
  std::vector<int32_t> retrieve;
  int32_t n_leaves = 0;
  for (int32_t i = 0; i < T; ++i) {
    if (has_child[i]) continue;
    retrieve.insert(retrieve.end(), path.begin() + static_cast<size_t>(i) * W,
                    path.begin() + static_cast<size_t>(i + 1) * W);
    ++n_leaves;
  }

  auto put = [&img](const void* src, size_t bytes) -> int64_t {
    int64_t off = align256(static_cast<int64_t>(img.size()));
    img.resize(static_cast<size_t>(off) + bytes, 0);
    if (bytes) std::memcpy(img.data() + off, src, bytes);
    return off;
  };
  d.T = T;
  d.D = D;
  d.n_leaves = n_leaves;
  d.pad = 0;
  d.off_parent = put(parent, T * sizeof(int32_t));
  d.off_depth = put(depth.data(), T * sizeof(int32_t));
  d.off_mask = put(mask.data(), mask.size() * sizeof(uint32_t));
  d.off_path = put(path.data(), path.size() * sizeof(int32_t));
  d.off_retrieve = put(retrieve.data(), retrieve.size() * sizeof(int32_t));
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

extern "C" const char* entmtp_last_error(void) { return g_last_error.c_str(); }

extern "C" const char* entmtp_version(void) { return "entmtp-gfx950 0.1"; }

extern "C" int32_t entmtp_bank_build(const int32_t* parents, const int32_t* sizes,
                                     int32_t n_trees, void* arena, size_t arena_bytes,
                                     size_t* arena_needed, void* stream, entmtp_bank** out) {
  clear_error();
  if (out) *out = nullptr;
  ENTMTP_CHECK_ARG(parents && sizes, ENTMTP_EINVAL, "parents and sizes must be non-NULL");
  ENTMTP_CHECK_ARG(n_trees >= 1, ENTMTP_EINVAL, "n_trees = %d < 1", n_trees);
  ENTMTP_CHECK_ARG(arena == nullptr || out != nullptr, ENTMTP_EINVAL,
                   "an upload needs an output handle");
  // validate every tree before planning any
  int64_t base = 0;
  for (int32_t t = 0; t < n_trees; ++t) {
    const int32_t T = sizes[t];
    ENTMTP_CHECK_ARG(T >= 1 && T <= ENTMTP_T_MAX, ENTMTP_ERANGE,
                     "tree %d: size %d outside [1, %d]", t, T, ENTMTP_T_MAX);
    const int32_t* p = parents + base;
    ENTMTP_CHECK_ARG(p[0] == -1, ENTMTP_ETREE, "tree %d: root parent is %d, not -1", t, p[0]);
    int32_t depth_max = 0;
    std::vector<int32_t> depth(T, 0);
    for (int32_t i = 1; i < T; ++i) {
      ENTMTP_CHECK_ARG(p[i] >= 0 && p[i] < i, ENTMTP_ETREE,
                       "tree %d: parent[%d] = %d is not an earlier node", t, i, p[i]);
      depth[i] = depth[p[i]] + 1;
      depth_max = depth[i] > depth_max ? depth[i] : depth_max;
    }
    ENTMTP_CHECK_ARG(depth_max <= ENTMTP_D_MAX, ENTMTP_ERANGE,
                     "tree %d: depth %d exceeds %d", t, depth_max, ENTMTP_D_MAX);
    base += T;
  }

  auto* bank = new entmtp_bank();
  bank->desc.resize(n_trees);
  base = 0;
  for (int32_t t = 0; t < n_trees; ++t) {
    plan_tree(parents + base, sizes[t], bank->image, bank->desc[t]);
    base += sizes[t];
  }
  bank->image.resize(static_cast<size_t>(align256(static_cast<int64_t>(bank->image.size()))), 0);
  const size_t need = bank->image.size();
  if (arena_needed) *arena_needed = need;

  if (arena == nullptr) {
    if (out) *out = bank;
    else delete bank;
    return ENTMTP_OK;
  }
  if (arena_bytes < need) {
    delete bank;
    return fail(ENTMTP_ENOSPC, "arena has %zu bytes, the bank needs %zu", arena_bytes, need);
  }
  auto s = static_cast<hipStream_t>(stream);
  int32_t rc = hip_status(hipGetDevice(&bank->device), "hipGetDevice");
  if (rc == ENTMTP_OK)
    rc = hip_status(hipMemcpyAsync(arena, bank->image.data(), need, hipMemcpyHostToDevice, s),
                    "bank upload");
  if (rc == ENTMTP_OK) rc = hip_status(hipStreamSynchronize(s), "bank upload sync");
  if (rc != ENTMTP_OK) {
    delete bank;
    return rc;
  }
  bank->arena = static_cast<uint8_t*>(arena);
  *out = bank;
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_bank_destroy(entmtp_bank* bank) {
  delete bank;
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_bank_size(const entmtp_bank* bank) {
  clear_error();
  ENTMTP_CHECK_ARG(bank != nullptr, ENTMTP_EINVAL, "bank is NULL");
  return static_cast<int32_t>(bank->desc.size());
}

extern "C" int32_t entmtp_bank_info(const entmtp_bank* bank, int32_t topo, int32_t* T,
                                    int32_t* D, int32_t* n_leaves) {
  clear_error();
  ENTMTP_CHECK_ARG(bank != nullptr, ENTMTP_EINVAL, "bank is NULL");
  ENTMTP_CHECK_ARG(topo >= 0 && topo < static_cast<int32_t>(bank->desc.size()), ENTMTP_EINVAL,
                   "topo %d outside [0, %zu)", topo, bank->desc.size());
  const TopoDesc& d = bank->desc[topo];
  if (T) *T = d.T;
  if (D) *D = d.D;
  if (n_leaves) *n_leaves = d.n_leaves;
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_bank_export(const entmtp_bank* bank, int32_t topo, uint32_t* mask,
                                      int32_t* depth, int32_t* path, int32_t* retrieve,
                                      int32_t* parent) {
  clear_error();
  ENTMTP_CHECK_ARG(bank != nullptr, ENTMTP_EINVAL, "bank is NULL");
  ENTMTP_CHECK_ARG(topo >= 0 && topo < static_cast<int32_t>(bank->desc.size()), ENTMTP_EINVAL,
                   "topo %d outside [0, %zu)", topo, bank->desc.size());
  const TopoDesc& d = bank->desc[topo];
  const uint8_t* img = bank->image.data();
  const size_t W = static_cast<size_t>(d.D) + 1;
  if (mask) std::memcpy(mask, img + d.off_mask, sizeof(uint32_t) * d.T * ENTMTP_MASK_WORDS);
  if (depth) std::memcpy(depth, img + d.off_depth, sizeof(int32_t) * d.T);
  if (path) std::memcpy(path, img + d.off_path, sizeof(int32_t) * d.T * W);
  if (retrieve) std::memcpy(retrieve, img + d.off_retrieve, sizeof(int32_t) * d.n_leaves * W);
  if (parent) std::memcpy(parent, img + d.off_parent, sizeof(int32_t) * d.T);
  return ENTMTP_OK;
}

extern "C" int32_t entmtp_ladder_next(int32_t rung, int32_t n_rungs, float s, float tau_on,
                                      float tau_off) {
  clear_error();
  ENTMTP_CHECK_ARG(n_rungs >= 1, ENTMTP_EINVAL, "n_rungs = %d < 1", n_rungs);
  ENTMTP_CHECK_ARG(rung >= 0 && rung < n_rungs, ENTMTP_EINVAL, "rung %d outside [0, %d)",
                   rung, n_rungs);
  ENTMTP_CHECK_ARG(tau_off <= tau_on, ENTMTP_EINVAL, "tau_off %g > tau_on %g",
                   static_cast<double>(tau_off), static_cast<double>(tau_on));
  return ladder_step(rung, n_rungs, s, tau_on, tau_off);
}

extern "C" int32_t entmtp_ladder_next_batched(int32_t B, int32_t* rung, const float* s,
                                              int32_t n_rungs, float tau_on, float tau_off) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 0, ENTMTP_EINVAL, "B = %d < 0", B);
  ENTMTP_CHECK_ARG(B == 0 || (rung && s), ENTMTP_EINVAL, "null rung or s array");
  ENTMTP_CHECK_ARG(n_rungs >= 1, ENTMTP_EINVAL, "n_rungs = %d < 1", n_rungs);
  ENTMTP_CHECK_ARG(tau_off <= tau_on, ENTMTP_EINVAL, "tau_off %g > tau_on %g",
                   static_cast<double>(tau_off), static_cast<double>(tau_on));
  for (int32_t b = 0; b < B; ++b)
    ENTMTP_CHECK_ARG(rung[b] >= 0 && rung[b] < n_rungs, ENTMTP_EINVAL,
                     "rung[%d] = %d outside [0, %d)", b, rung[b], n_rungs);
  for (int32_t b = 0; b < B; ++b) rung[b] = ladder_step(rung[b], n_rungs, s[b], tau_on, tau_off);
  return ENTMTP_OK;
}

// NextChildren(T, D) of Algorithm 1 and the joint tree T u F built from it:
// a node's next-ranked child hangs under it, so each node of depth below D
// contributes exactly one candidate, appended in node order.
extern "C" int32_t entmtp_frontier_tree(const int32_t* parent, int32_t T, int32_t max_depth,
                                        int32_t* joint_parent, uint8_t* in_tree,
                                        int32_t joint_capacity, int32_t* joint_T) {
  clear_error();
  ENTMTP_CHECK_ARG(parent && joint_parent && joint_T, ENTMTP_EINVAL,
                   "parent, joint_parent and joint_T must be non-NULL");
  ENTMTP_CHECK_ARG(T >= 1, ENTMTP_EINVAL, "T = %d < 1", T);
  ENTMTP_CHECK_ARG(max_depth >= 0, ENTMTP_EINVAL, "max_depth = %d < 0", max_depth);
  ENTMTP_CHECK_ARG(parent[0] == -1, ENTMTP_EINVAL, "parent[0] = %d, the root's must be -1", parent[0]);
  std::vector<int32_t> depth(static_cast<size_t>(T), 0);
  int32_t n_cand = 0;
  for (int32_t i = 0; i < T; ++i) {
    if (i > 0) {
      ENTMTP_CHECK_ARG(parent[i] >= 0 && parent[i] < i, ENTMTP_EINVAL,
                       "parent[%d] = %d: parents must precede their children", i, parent[i]);
      depth[i] = depth[parent[i]] + 1;
    }
    n_cand += depth[i] < max_depth ? 1 : 0;
  }
  *joint_T = T + n_cand;
  ENTMTP_CHECK_ARG(T + n_cand <= joint_capacity, ENTMTP_ENOSPC,
                   "joint tree has %d nodes, capacity %d", T + n_cand, joint_capacity);
  int32_t k = T;
  for (int32_t i = 0; i < T; ++i) {
    joint_parent[i] = parent[i];
    if (in_tree) in_tree[i] = 1u;
    if (depth[i] < max_depth) {
      joint_parent[k] = i;
      if (in_tree) in_tree[k] = 0u;
      ++k;
    }
  }
  return ENTMTP_OK;
}
