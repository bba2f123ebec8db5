// LM-head verification logits: logits[i][v] = sum_k X[i][k] * W[v][k].
//
// The verification pass of §2.3 scores every draft-tree node with the
// target's LM head (the next-token distribution softmax(W h) of §2.2).  At
// batch 1 the tree has tens of nodes, so the product is a skinny GEMM whose
// cost is streaming W (V x hid bf16, 262 MB for a 7B vocabulary) once from
// HBM; the arithmetic intensity is about T flop per byte.
//
// Design (gfx950):
//  * W rows are the MFMA M dimension and tree nodes the N dimension of
//    v_mfma_f32_16x16x32_bf16.  Each lane loads its A operand straight from
//    HBM into registers: lane (row r = lane%16, group g = lane/16) reads 16
//    bytes of row r at k = 32s + 8g for step s, so a wave instruction covers
//    16 rows x 64 contiguous bytes.  W is never staged in LDS.
//  * X (the tree's hidden states) is shared by every W row: each workgroup
//    stages a K-chunk of X in LDS (double buffered, row padding against bank
//    conflicts) and every wave reads its B operands from there.
//  * The vocabulary is cut into one contiguous slice per workgroup, sized so
//    every CU streams the same number of bytes; inside the slice the 16-row
//    tiles are dealt round-robin to the four waves (at most two each).
//  * The next K-chunk of W and X is loaded while the current one is
//    multiplied, so each wave keeps two chunks of loads in flight.
//  * Accumulation is fp32; logits are written as fp32 so that the argmax and
//    the statistics never see a rounded logit.
#include "common.hpp"

namespace entmtp {
namespace {

constexpr int kLmThreads = 256;
constexpr int kLmWaves = kLmThreads / 64;
constexpr int kLmTiles = 2;                         // 16-row tiles per wave
constexpr int kLmRowsPerBlock = 16 * kLmTiles * kLmWaves;  // 128

__device__ __forceinline__ int slice_begin(int b, int G, int V) {
  if (b >= G) return V;
  return static_cast<int>((static_cast<long long>(V) * b / G) & ~3ll);
}

template <int NT, int BK>
__global__ __launch_bounds__(kLmThreads) void lm_head_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    int T, int hid, int V, int G) {
  constexpr int TP = NT * 16;      // node rows per pass
  constexpr int STEPS = BK / 32;   // MFMA k-steps per chunk
  constexpr int LDX = BK + 8;      // LDS row stride in bf16 (16-byte pad)
  constexpr int XU = TP * BK / 8;  // 16-byte units of one X chunk
  constexpr int XU_PER_THREAD = (XU + kLmThreads - 1) / kLmThreads;
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][TP * LDX];

  const int r0 = slice_begin(blockIdx.x, G, V);
  const int r1 = slice_begin(blockIdx.x + 1, G, V);
  const int j0 = blockIdx.y * TP;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;

  const uint16_t* wrow[kLmTiles];
  bool wok[kLmTiles], live[kLmTiles];
#pragma unroll
  for (int t = 0; t < kLmTiles; ++t) {
    const int tb = r0 + 16 * (wave + kLmWaves * t);
    live[t] = tb < r1;
    wok[t] = tb + lr < r1;
    wrow[t] = W + static_cast<size_t>(wok[t] ? tb + lr : 0) * hid + 8 * lg;
  }

  auto load_w = [&](u32x4 (&a)[kLmTiles][STEPS], int kc) {
#pragma unroll
    for (int t = 0; t < kLmTiles; ++t)
#pragma unroll
      for (int s = 0; s < STEPS; ++s) {
        const int k = kc + 32 * s;
        a[t][s] = (wok[t] && k + 8 * lg < hid)
                      ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wrow[t] + k))
                      : u32x4{0u, 0u, 0u, 0u};
      }
  };
  auto load_x = [&](u32x4 (&x)[XU_PER_THREAD], int kc) {
#pragma unroll
    for (int q = 0; q < XU_PER_THREAD; ++q) {
      const int u = tid + q * kLmThreads;
      const int j = u / (BK / 8), c8 = u % (BK / 8);
      const int node = j0 + j, k = kc + 8 * c8;
      x[q] = (u < XU && node < T && k < hid)
                 ? *reinterpret_cast<const u32x4*>(X + static_cast<size_t>(node) * hid + k)
                 : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_x = [&](const u32x4 (&x)[XU_PER_THREAD], int buf) {
#pragma unroll
    for (int q = 0; q < XU_PER_THREAD; ++q) {
      const int u = tid + q * kLmThreads;
      if (u < XU) {
        const int j = u / (BK / 8), c8 = u % (BK / 8);
        *reinterpret_cast<u32x4*>(&xs[buf][j * LDX + 8 * c8]) = x[q];
      }
    }
  };

  f32x4 acc[kLmTiles][NT];
#pragma unroll
  for (int t = 0; t < kLmTiles; ++t)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[t][n] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto mma_chunk = [&](const u32x4 (&a)[kLmTiles][STEPS], int buf) {
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      bf16x8 b[NT];
#pragma unroll
      for (int n = 0; n < NT; ++n)
        b[n] = as_bf16x8(*reinterpret_cast<const u32x4*>(&xs[buf][(n * 16 + lr) * LDX + 32 * s + 8 * lg]));
#pragma unroll
      for (int t = 0; t < kLmTiles; ++t) {
        if (!live[t]) continue;
        const bf16x8 av = as_bf16x8(a[t][s]);
#pragma unroll
        for (int n = 0; n < NT; ++n)
          acc[t][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, b[n], acc[t][n], 0, 0, 0);
      }
    }
  };

  const int nchunks = (hid + BK - 1) / BK;
  u32x4 a0[kLmTiles][STEPS], a1[kLmTiles][STEPS];
  u32x4 xr[XU_PER_THREAD];
  load_x(xr, 0);
  load_w(a0, 0);
  store_x(xr, 0);
  for (int c = 0; c < nchunks; c += 2) {
    // even chunk: multiply a0 / xs[0] while a1 / xs[1] arrive
    __syncthreads();
    const bool more1 = c + 1 < nchunks;
    if (more1) {
      load_x(xr, (c + 1) * BK);
      load_w(a1, (c + 1) * BK);
    }
    mma_chunk(a0, 0);
    if (more1) store_x(xr, 1);
    if (!more1) break;
    // odd chunk
    __syncthreads();
    const bool more2 = c + 2 < nchunks;
    if (more2) {
      load_x(xr, (c + 2) * BK);
      load_w(a0, (c + 2) * BK);
    }
    mma_chunk(a1, 1);
    if (more2) store_x(xr, 0);
  }

  // epilogue: lane holds rows 4*lg..4*lg+3 of each tile for node column lr
  const bool vec_ok = (V & 3) == 0;
#pragma unroll
  for (int t = 0; t < kLmTiles; ++t) {
    if (!live[t]) continue;
    const int v = r0 + 16 * (wave + kLmWaves * t) + 4 * lg;
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      const int node = j0 + n * 16 + lr;
      if (node >= T) continue;
      float* dst = logits + static_cast<size_t>(node) * V + v;
      if (vec_ok && v + 3 < r1) {
        *reinterpret_cast<f32x4*>(dst) = acc[t][n];
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (v + r < r1) dst[r] = acc[t][n][r];
      }
    }
  }
}

template <int NT, int BK>
int32_t launch_lm(const uint16_t* X, const uint16_t* W, float* logits, int T, int hid, int V,
                  hipStream_t s) {
  // one slice per workgroup, at most kLmRowsPerBlock rows, at least one per CU
  const int want = (V + kLmRowsPerBlock - 5) / (kLmRowsPerBlock - 4);
  int G = want > 256 ? want : 256;
  const int max_g = (V + 3) / 4;
  G = G < max_g ? G : max_g;
  const int passes = (T + NT * 16 - 1) / (NT * 16);
  hipLaunchKernelGGL((lm_head_kernel<NT, BK>), dim3(G, passes), dim3(kLmThreads), 0, s, X, W,
                     logits, T, hid, V, G);
  return launch_status("verify_logits launch");
}

}  // namespace
}  // namespace entmtp

using namespace entmtp;

extern "C" int32_t entmtp_verify_logits(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                        int32_t T, int32_t hid, int32_t V, float* logits,
                                        void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(hidden && w_lm && logits, ENTMTP_EINVAL, "hidden, w_lm, logits must be non-NULL");
  ENTMTP_CHECK_ARG(T >= 1 && T <= 4096, ENTMTP_EINVAL, "T = %d outside [1, 4096]", T);
  ENTMTP_CHECK_ARG(hid >= 8 && hid % 8 == 0, ENTMTP_EINVAL, "hid = %d must be a positive multiple of 8", hid);
  ENTMTP_CHECK_ARG(V >= 1, ENTMTP_EINVAL, "V = %d < 1", V);
  ENTMTP_CHECK_ARG(aligned16(hidden) && aligned16(w_lm) && aligned16(logits), ENTMTP_EINVAL,
                   "hidden, w_lm and logits must be 16-byte aligned");
  auto s = static_cast<hipStream_t>(stream);
  if (T <= 16) return launch_lm<1, 256>(hidden, w_lm, logits, T, hid, V, s);
  if (T <= 32) return launch_lm<2, 256>(hidden, w_lm, logits, T, hid, V, s);
  if (T <= 64) return launch_lm<4, 128>(hidden, w_lm, logits, T, hid, V, s);
  return launch_lm<8, 128>(hidden, w_lm, logits, T, hid, V, s);
}
