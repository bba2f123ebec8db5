// Internal definitions shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "entmtp.h"

namespace entmtp {

// ---------------------------------------------------------------- errors --

// Records `msg` as the calling thread's last error and returns `code`.
int32_t fail(int32_t code, const char* fmt, ...);
void clear_error();

#define ENTMTP_CHECK_ARG(cond, code, ...) \
  do {                                    \
    if (!(cond)) return ::entmtp::fail(code, __VA_ARGS__); \
  } while (0)

// Checks the launch that was just made (or any HIP call's return code).
int32_t hip_status(hipError_t e, const char* what);
inline int32_t launch_status(const char* what) { return hip_status(hipGetLastError(), what); }

// ------------------------------------------------------------------ bank --

// Byte offsets of one tree's arrays inside the bank arena.
struct TopoDesc {
  int32_t T;         // nodes, root included
  int32_t D;         // depth of the deepest node
  int32_t n_leaves;
  int32_t pad;
  int64_t off_parent;    // int32[T]
  int64_t off_depth;     // int32[T]
  int64_t off_mask;      // uint32[T][ENTMTP_MASK_WORDS]
  int64_t off_path;      // int32[T][D+1]
  int64_t off_retrieve;  // int32[n_leaves][D+1]
};

}  // namespace entmtp

struct entmtp_bank {
  std::vector<entmtp::TopoDesc> desc;
  std::vector<uint8_t> image;  // host copy of the arena contents
  uint8_t* arena = nullptr;    // device arena (nullptr for a host-only bank)
  int device = -1;
};

namespace entmtp {

// Validates (bank, topo) for a kernel launch; returns 0 or an error status.
int32_t check_device_bank(const entmtp_bank* bank, int32_t topo);

// Device-side state of a decode loop whose tree choice runs on the GPU (§4's
// policy moved next to the statistics it reads): one slot per step parity,
// the step with parity p reads slot p and its acceptance writes slot p ^ 1.
struct DevStep {
  int rung;      // bank index of the step's tree
  int T;         // its node count
  int L;         // prefix length
  int step;      // steps since the device state was started
  int overflow;  // sticky: a step's prefix plus tree exceeded the cache (no attention since)
};

// A bank tree as the device-scheduled kernels find it: sizes and byte
// offsets of its arrays in the bank arena.
struct DevTopo {
  int T, D;
  int off_parent, off_depth, off_mask, off_path;
  int pad[2];
  // attention split count for this tree by split bound (index 1..32; the
  // lone-sequence choice depends on the prefix length only through it)
  unsigned char splits[36];
};

// The hysteretic ladder of §4 over a bank sorted by size: climb one rung when
// s > tau_on, descend one when s <= tau_off, else stay (clamped to the bank).
__host__ __device__ inline int ladder_step(int rung, int n_rungs, float s, float tau_on,
                                           float tau_off) {
  if (s > tau_on) return rung + 1 < n_rungs ? rung + 1 : rung;
  if (s <= tau_off) return rung > 0 ? rung - 1 : 0;
  return rung;
}

// Grids of the attention for a tree chosen on the device: sized for the
// largest plan any bank tree can need at prefix lengths up to cap - T.
struct DevAttnShape {
  int rows = 0, merge_blocks = 0, T_max = 0, D_max = 0;
  int items[5] = {0, 0, 0, 0, 0};   // attend workgroups of the instance with 1 / 2 / 4 query tiles
  size_t need = 0;   // workspace bytes
};

int32_t attn_device_shape(const entmtp_bank* bank, int Hq, int Hkv, int cap, DevAttnShape* out);

// Fills DevTopo::splits of every bank tree for the current device.
void attn_device_splits(const entmtp_bank* bank, int Hq, int Hkv, DevTopo* topos);

// One attention layer (as entmtp_tree_attn) for the tree and prefix length
// held in *dev; topos is the bank's device descriptor table.
int32_t launch_attn_device(const entmtp_bank* bank, const DevStep* dev, const DevTopo* topos,
                           const DevAttnShape& sh, const entmtp_bf16* q, const entmtp_bf16* k_tree,
                           const entmtp_bf16* v_tree, entmtp_bf16* k_cache, entmtp_bf16* v_cache,
                           int cap, int Hq, int Hkv, float scale, float rope_theta,
                           entmtp_bf16* out, void* workspace, hipStream_t stream);

// Result of one verification step as the host reads it, written by the accept
// kernel into coherent pinned host memory.  Every word is 64 bits: the step's
// sequence number in the upper half and one field in the lower half, stored
// by one lane as a single system-scope store.  A word is therefore complete
// or stale, never torn, and the host takes the record once every word it
// needs carries the sequence number it waits for -- no fence orders the
// words, so publishing costs the kernel no cache write-back.
constexpr int kMirrorPathWords = (ENTMTP_D_MAX + 1 + 3) / 4;  // 4 path entries per word
constexpr int kMirrorWords = 3 + kMirrorPathWords;
struct StepMirror {
  uint64_t accept_len;
  uint64_t bonus;
  uint64_t best_top1p;                  // float bits
  uint64_t path[kMirrorPathWords];      // node index bytes, entry j in byte j % 4 of word j / 4
};
static_assert(sizeof(StepMirror) == kMirrorWords * sizeof(uint64_t), "mirror layout");

// Launches the accept kernel (no argument checks beyond the bank's); with a
// non-NULL `mirror` (device address of host memory) it also publishes the
// result there under sequence number `seq`.
// path_capacity entries of `path` are written (-1 past the accept length);
// at least the tree's depth + 1, at most ENTMTP_D_MAX + 1.
int32_t launch_accept(const entmtp_bank* bank, int32_t topo, const int32_t* draft_tokens,
                      const int32_t* argmax, const float* top1p, int32_t* accept_len,
                      int32_t* path, int32_t path_capacity, int32_t* bonus, float* best_top1p,
                      StepMirror* mirror, uint32_t seq, hipStream_t stream);

// The device-scheduled form: the tree is bank entry cur->rung; the drafts of
// bank tree k are row k of drafts [n_topo][tree_rows]; after accepting, the
// ladder picks the next tree from s = top1p[best] and writes *next =
// {rung', T', L + accept_len + 1}; log (4 ints, may be NULL) receives
// (rung, L, accept_len, s bits) in row cur->step % log_rows of a
// [log_rows][4] array; user_accept_len / user_path (may be NULL) receive
// copies of the accept length and path.  prefix_fixed: the next step keeps
// prefix length L (every step verifies at the same position).  A step whose
// L + T exceeds cap (its attention computed nothing) sets the sticky overflow
// flag: from then on the prefix and tree stay where they are and the log
// records accept length -1.
struct FinAccDevice {
  const DevStep* cur;
  DevStep* next;
  const DevTopo* topos;
  const int32_t* drafts;
  int32_t tree_rows, n_topo;
  int32_t cap, prefix_fixed;
  float tau_on, tau_off;
  int32_t* log;
  int32_t log_rows;
  int32_t* user_accept_len;
  int32_t* user_path;
};
int32_t launch_finalize_accept_device(const entmtp_bank* bank, const FinAccDevice& dv,
                                      const void* partials, int32_t V, float inv_temp,
                                      float* entropy, float* top1p, int32_t* argmax,
                                      int32_t* accept_len, int32_t* path, int32_t path_capacity,
                                      int32_t* bonus, float* best_top1p, StepMirror* mirror,
                                      uint32_t seq, hipStream_t stream);

// Compaction (as entmtp_kv_compact, one sequence) at the prefix length dev->L.
int32_t launch_compact_device(const DevStep* dev, const int32_t* path, int32_t path_capacity,
                              const int32_t* accept_len, entmtp_bf16* k_cache,
                              entmtp_bf16* v_cache, int32_t n_layers, int64_t layer_stride,
                              int32_t Hkv, int32_t cap, int32_t d, hipStream_t s);

// Compaction (as entmtp_kv_compact, one sequence) of a path the host already
// holds: path_host[0..accept_len] travels in the launch's arguments, so the
// kernel reads no device result (0 <= accept_len <= ENTMTP_D_MAX).
int32_t launch_compact_host(const int32_t* path_host, int32_t accept_len, int32_t prefix_len,
                            entmtp_bf16* k_cache, entmtp_bf16* v_cache, int32_t n_layers,
                            int64_t layer_stride, int32_t Hkv, int32_t cap, int32_t d,
                            hipStream_t s);

// Finishes the LM head's statistics partials for every node of tree `topo`
// (n_parts partials per node, rows n_parts long: what the LM head launched
// for the step wrote) and accepts the tree (as launch_accept): one launch
// for trees of up to 32 nodes, a statistics launch and an acceptance launch
// for larger ones.
int32_t launch_finalize_accept(const entmtp_bank* bank, int32_t topo, const void* partials,
                               int32_t n_parts, int32_t V, float inv_temp, float* entropy,
                               float* top1p,
                               int32_t* argmax, const int32_t* draft_tokens, int32_t* accept_len,
                               int32_t* path, int32_t path_capacity, int32_t* bonus,
                               float* best_top1p, StepMirror* mirror, uint32_t seq,
                               hipStream_t stream);

template <typename T>
inline const T* bank_ptr(const entmtp_bank* b, int64_t off) {
  return reinterpret_cast<const T*>(b->arena + off);
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// --------------------------------------------------------- device helpers --

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// fp64 -> bf16 bits with a single rounding (nearest even) straight from the
// double's mantissa: after rounding the mantissa to 7 bits the value is
// exactly representable in fp32, whose top half is the bf16 pattern.
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double x) {
  uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  const uint64_t lsb = (u >> 45) & 1ull;
  u += 0x00000FFFFFFFFFFFull + lsb;
  u &= ~0x00001FFFFFFFFFFFull;
  float f = static_cast<float>(__longlong_as_double(static_cast<long long>(u)));
  return __float_as_uint(f) >> 16;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ double bf16_to_f64(uint16_t b) {
  return static_cast<double>(__uint_as_float(static_cast<uint32_t>(b) << 16));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

}  // namespace entmtp
