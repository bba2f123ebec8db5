// LM-head verification logits: logits[i][v] = sum_k X[i][k] * W[v][k], and
// the per-node softmax statistics taken from the same accumulators.
//
// The verification pass of §2.3 scores every draft-tree node with the
// target's LM head (the next-token distribution softmax(W h) of §2.2).  At
// batch 1 the tree has tens of nodes, so the product is a skinny GEMM whose
// cost is streaming W (V x hid bf16, 262 MB for a 7B vocabulary) once from
// HBM; the arithmetic intensity is about T flop per byte.
//
// The streaming kernel (hyb_body; hid a multiple of 512), on
// v_mfma_f32_16x16x32_bf16 with W rows as M and tree nodes as N:
//  * the vocabulary is cut into slices of at most 64 rows, one per workgroup
//    of four waves, and the grid is a whole multiple of the CU count (a
//    partial extra round of workgroups costs ~20%);
//  * each wave streams its own 16-row W tile through VGPRs, 4 rows x 256
//    contiguous bytes per load instruction, several K-stages deep, and turns
//    each stage into MFMA operand layout through a private XOR-swizzled LDS
//    tile;
//  * X, shared by all waves, arrives by direct global->LDS copies into a ring
//    of separate LDS objects (one per stage, so the compiler can tell the
//    slot being read from the slots in flight), one barrier per stage;
//  * loads are unconditional (clamped rows) and the K loop is unrolled
//    completely for hid 4096 / 5120, so the explicit wait counts stay exact;
//  * workgroups walk K in rotated order;
//  * with statistics, the epilogue reduces each node's accumulators over the
//    slice to a partial (raw max and its index, sum e^(y-m), sum (y-m)e^(y-m))
//    through wave shuffles and the wave's own transposition tile, and a small
//    kernel merges a node's partials (stats.hpp), so logits never need to
//    reach memory.
//  * each k-step's A and B fragments are read from LDS one step ahead of
//    their products, so the LDS latency hides behind the MFMAs;
//  * 64- and 128-node tiles give each wave two 16-row W tiles (a workgroup
//    takes two consecutive slices), so every X fragment read from LDS feeds
//    two products.
// Node tiles of 16, 32, 64 or 128 nodes select the instantiation; variants
// loop a workgroup over several slices (one workgroup per CU, leaving room for
// concurrent attention) or read the node count from device memory (trees
// chosen on the GPU).  Other hidden sizes use a direct-to-LDS kernel
// (hid % 128 == 0) or a register-prefetch kernel.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "stats.hpp"
#include "stream_pipe.hpp"

namespace entmtp {
namespace {

constexpr int kLmThreads = 256;
constexpr int kLmWaves = kLmThreads / 64;
constexpr int kLmTiles = 2;                         // 16-row tiles per wave
constexpr int kLmRowsPerBlock = 16 * kLmTiles * kLmWaves;  // 128

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

// ---------------------------------------------------------------------------
// Streaming variant for hid % 128 == 0: W and X reach LDS through direct
// global->LDS loads (global_load_lds_dwordx4), which keep several K-stages in
// flight without holding them in VGPRs.  Each of the eight waves owns one
// 16-row W tile and a private ring of S stages (16 rows x 128 k = 4 KB each);
// the X stage (16*NT nodes x 128 k) is shared by the workgroup.  A load
// instruction covers 4 rows x 256 contiguous bytes; lane p of a row fetches
// chunk p ^ row, so the MFMA-layout reads (16 rows, same chunk) hit 16
// different bank groups.  One barrier per stage; S-1 stages stay in flight.
// ---------------------------------------------------------------------------
constexpr int kL3Waves = 8;
constexpr int kL3Threads = 64 * kL3Waves;
constexpr int kL3Bk = 128;                 // k per stage
constexpr int kL3RowBytes = kL3Bk * 2;     // 256
constexpr int kL3TileBytes = 16 * kL3RowBytes;

template <int NT>
struct L3Shape {
  static constexpr int TP = 16 * NT;                      // node rows per pass
  static constexpr int RPI = 4;                           // X rows per load instruction
  static constexpr int NXI = TP / RPI;                    // distinct X instructions per stage
  static constexpr int XI = NXI >= kL3Waves ? NXI / kL3Waves : 1;   // per wave
  static constexpr int PER_STAGE = 4 + XI;                // loads per wave per stage
  static constexpr int XOFF = kL3Waves * kL3TileBytes;    // X stage after the eight W tiles
  static constexpr int SLOT = XOFF + TP * kL3RowBytes;    // bytes per ring slot
  static_assert(NXI % kL3Waves == 0 || NXI < kL3Waves, "X split");
};

template <int NT, int S>
__global__ __launch_bounds__(kL3Threads) void lm_head_lds_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    int T, int hid, int V, int G) {
  using Sh = L3Shape<NT>;
  static_assert(S >= 2 && S <= 4, "2 to 4 stages");
  // ring slot k lives at ring + k * SLOT; every access uses a compile-time
  // slot offset, so the compiler can tell the slot being read from the slots
  // that loads in flight write to
  __shared__ __attribute__((aligned(16))) uint8_t ring[S * Sh::SLOT];

  const int r0 = slice_begin(blockIdx.x, G, V);
  const int r1 = slice_begin(blockIdx.x + 1, G, V);
  if (r0 >= r1) return;  // empty slice (tiny V): the whole workgroup leaves
  const int j0 = blockIdx.y * Sh::TP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int tile0 = r0 + 16 * wave;
  const bool live = tile0 < r1;

  // Per-lane source pointers (row, swizzled chunk).  Every wave issues
  // exactly PER_STAGE loads per stage -- the explicit vmcnt waits count on
  // it -- so lanes of rows past the slice or past T read an in-bounds row
  // this wave loads anyway (an L2 hit) instead of being masked off; the
  // results of those rows and columns are never stored.
  const uint16_t* wsrc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = 4 * i + (lane >> 4);
    const int row = tile0 + rr < r1 ? tile0 + rr : (live ? tile0 : r0);
    wsrc[i] = W + static_cast<size_t>(row) * hid + 8 * ((lane & 15) ^ rr);
  }
  // X: instruction n fills rows 4n..4n+3 of the stage.  With fewer distinct
  // instructions than waves (NT = 1) the extra waves repeat one: identical
  // bytes to identical addresses, and every wave keeps the same load count.
  const uint16_t* xsrc[Sh::XI];
  int xoff[Sh::XI];
#pragma unroll
  for (int q = 0; q < Sh::XI; ++q) {
    const int n = (wave * Sh::XI + q) % Sh::NXI;
    const int rr = n * Sh::RPI + (lane >> 4);   // X row written by this lane
    const int node = j0 + rr < T ? j0 + rr : j0;
    xsrc[q] = X + static_cast<size_t>(node) * hid + 8 * ((lane & 15) ^ (rr & 15));
    xoff[q] = Sh::XOFF + n * Sh::RPI * kL3RowBytes;
  }

  // Workgroups walk K in rotated order (start stage differs per workgroup):
  // otherwise every CU streams the same column band of its rows at the same
  // time, and accesses 8 KB apart pile onto the same HBM channels.
  const int nch = hid / kL3Bk;
  const int rot = static_cast<int>((static_cast<unsigned>(blockIdx.x) * 7u) % static_cast<unsigned>(nch));
  auto issue = [&](uint8_t* base, int stage) {
    int ks = stage + rot;
    ks = ks >= nch ? ks - nch : ks;
    const int koff = ks * kL3Bk;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      lds_dma16(wsrc[i] + koff, base + wave * kL3TileBytes + i * 1024);
#pragma unroll
    for (int q = 0; q < Sh::XI; ++q)
      lds_dma16(xsrc[q] + koff, base + xoff[q]);
  };

  f32x4 acc[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const uint8_t* base) {
    const uint8_t* wt = base + wave * kL3TileBytes;
    const uint8_t* xt = base + Sh::XOFF;
#pragma unroll
    for (int s = 0; s < kL3Bk / 32; ++s) {
      const int ch = 4 * s + lg;
      const bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4*>(wt + lr * kL3RowBytes + ((ch ^ lr) << 4)));
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const bf16x8 b = as_bf16x8(*reinterpret_cast<const u32x4*>(
            xt + (n * 16 + lr) * kL3RowBytes + ((ch ^ lr) << 4)));
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[n], 0, 0, 0);
      }
    }
  };

  // One pipeline step: wait for stage c, barrier, refill the slot freed by
  // stage c-1 with stage c+S-1, multiply stage c.  Loads are issued
  // unconditionally (past the last stage the index is clamped and the last
  // stage is fetched again), so after stage c exactly S-2 stages are always
  // in flight and the wait is exact; the compiler sees one load count on
  // every path and adds no drain of its own.
  auto step = [&](const uint8_t* cur, uint8_t* refill, int c) {
    wait_vmcnt<(S - 2) * Sh::PER_STAGE>();
    stage_barrier();
    issue(refill, c + S - 1 < nch ? c + S - 1 : nch - 1);
    if (live && c < nch) compute(cur);
  };
  constexpr int SL = Sh::SLOT;
  issue(ring, 0);
  if constexpr (S > 2) issue(ring + SL, 1 < nch ? 1 : nch - 1);
  if constexpr (S > 3) issue(ring + 2 * SL, 2 < nch ? 2 : nch - 1);
  for (int c = 0; c < nch; c += S) {
    step(ring, ring + ((S - 1) % S) * SL, c);
    step(ring + SL, ring + (S % S) * SL, c + 1);
    if constexpr (S > 2) step(ring + 2 * SL, ring + ((S + 1) % S) * SL, c + 2);
    if constexpr (S > 3) step(ring + 3 * SL, ring + ((S + 2) % S) * SL, c + 3);
  }
  wait_vmcnt<0>();   // no load may land in LDS after the workgroup is gone

  if (!live) return;
  const bool vec_ok = (V & 3) == 0;
  const int v = tile0 + 4 * lg;
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const int node = j0 + n * 16 + lr;
    if (node >= T) continue;
    float* dst = logits + static_cast<size_t>(node) * V + v;
    if (vec_ok && v + 3 < r1) {
      *reinterpret_cast<f32x4*>(dst) = acc[n];
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (v + r < r1) dst[r] = acc[n][r];
    }
  }
}

// ---------------------------------------------------------------------------
// Hybrid streaming variant (hid % 128 == 0): W through VGPRs, X through LDS.
// W is the byte stream: each wave keeps S K-stages of its 16-row tile in
// flight as plain VGPR loads (4 rows x 256 contiguous bytes per
// instruction -- the fastest read path measured on MI355X) and transposes
// each stage to MFMA operand layout through a private 4 KB LDS tile (lane p
// of row r stores chunk p at slot p ^ r: conflict-free both ways).  X, the
// same for every wave, arrives by direct global->LDS copies into a ring of S
// shared stages.  A stage's X copy is issued just before the stage's W loads;
// loads complete in order, so the wait the compiler places for the W
// registers also covers the X copy, and one barrier per stage publishes
// every wave's share.  All loads are issued unconditionally (addresses are
// clamped) so that every path carries the same load count.
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Softmax-statistics partials fused into the LM-head epilogue.  A partial of
// a set of vocabulary rows is (zmax, idx, Z, S): the largest raw logit and the
// lowest index attaining it (the argmax is decided on raw fp32 logits), and,
// with y = inv_temp * z and m = inv_temp * zmax, Z = sum e^(y - m) and
// S = sum (y - m) e^(y - m).  Partials merge exactly (up to rounding) after
// rescaling to the larger maximum, so the per-workgroup partials of every
// vocabulary slice combine into the row's entropy ln Z - S/Z, top-1
// probability 1/Z and argmax.
// ---------------------------------------------------------------------------
constexpr int kHybWaves = 4;                        // 64 rows per workgroup slice
// 64- and 128-node tiles: two W tiles per wave (slices paired per
// workgroup), X ring depth 4 and 2 (the 128-node X stage is 32 KB)
constexpr int kHybW4 = 2, kHybS4 = 4, kHybW8 = 2, kHybS8 = 2;
constexpr int kHybThreads = 64 * kHybWaves;

// X stage split for the hybrid kernel (four waves share the copies)
template <int NT>
struct HybShape {
  static constexpr int TP = 16 * NT;
  static constexpr int RPI = 4;
  static constexpr int NXI = TP / RPI;
  static constexpr int XI = NXI >= kHybWaves ? NXI / kHybWaves : 1;
  static_assert(NXI % kHybWaves == 0, "X split");
};

// The body of the streaming LM-head kernel for node tile NT (16 * NT nodes per
// pass, starting at node j0).  The kernels that call it own the LDS: one
// object per X ring slot, so that the compiler can tell the slot being read
// from the slots the copies in flight write to (the body is inlined, so the
// slots stay distinct objects), and the per-wave transposition tiles.
// Precondition (host dispatch): hid is a multiple of S * 128, and equals
// NCH * 128 when NCH > 0 (the K loop is then unrolled completely: no
// loop-carried stage registers, so the compiler's load bookkeeping stays
// exact and it never drains the pipeline).
template <int NT, int S, int NCH, bool STATS, int WT = 1>
__device__ __forceinline__ void hyb_body(uint8_t* xslot0, uint8_t* xslot1, uint8_t* xslot2,
                                         uint8_t* xslot3, uint8_t* tpose,
                                         const uint16_t* __restrict__ X,
                                         const uint16_t* __restrict__ W, float* __restrict__ logits,
                                         int T, int hid, int V, int G, float inv_temp,
                                         StatPart* __restrict__ part, int j0, int sl,
                                         int pcol = -1, int pstride = 0, bool merge_prev = false) {
  using Sh = HybShape<NT>;
  static_assert(S >= 2 && S <= 4, "two to four X ring slots");
  static_assert(WT == 1 || WT == 2, "one or two W tiles per wave");
  uint8_t* const xring[4] = {xslot0, xslot1, xslot2, xslot3};

  // a workgroup takes WT consecutive slices (sl is the first slice / WT)
  const int r0 = slice_begin(WT * sl, G, V);
  const int r1 = slice_begin(WT * sl + WT, G, V);
  if (r0 >= r1) {  // empty slices (tiny V): the whole workgroup leaves
    if constexpr (STATS)
      if (threadIdx.x < Sh::TP && j0 + threadIdx.x < T) {
        const StatPart empty{-INFINITY, 0.f, 0.f, 0x7fffffff};
        if (pcol >= 0) {
          if (!merge_prev) part[static_cast<size_t>(j0 + threadIdx.x) * pstride + pcol] = empty;
        } else {
#pragma unroll
          for (int u = 0; u < WT; ++u)
            part[static_cast<size_t>(j0 + threadIdx.x) * G + WT * sl + u] = empty;
        }
      }
    return;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  // wave w owns the 16-row tiles w, w + 4 (when WT = 2) of the rows [r0, r1)
  int tile0[WT];
  bool live[WT];
#pragma unroll
  for (int t = 0; t < WT; ++t) {
    tile0[t] = r0 + 16 * (wave + kHybWaves * t);
    live[t] = tile0[t] < r1;
  }
  const int nch = NCH > 0 ? NCH : hid / kL3Bk;
  // workgroups walk K in rotated order so that CUs do not all stream the
  // same column band at once
  const int rot = static_cast<int>((static_cast<unsigned>(sl) * 7u) % static_cast<unsigned>(nch));

  // W: instruction i, lane l -> row 4i + l/16, chunk l%16 (rows past the
  // slice read an in-bounds row of this slice; their outputs are not stored)
  const uint16_t* wsrc[WT][4];
#pragma unroll
  for (int t = 0; t < WT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = 4 * i + (lane >> 4);
      const int row = tile0[t] + rr < r1 ? tile0[t] + rr : (live[t] ? tile0[t] : r0);
      wsrc[t][i] = W + static_cast<size_t>(row) * hid + 8 * (lane & 15);
    }
  // X: copy instruction n fills stage rows 4n..4n+3, lane p of row r fetching
  // chunk p ^ r; with fewer distinct instructions than waves (NT = 1) extra
  // waves repeat one (identical bytes to identical addresses)
  const uint16_t* xsrc[Sh::XI];
  int xoff[Sh::XI];
#pragma unroll
  for (int q = 0; q < Sh::XI; ++q) {
    const int n = (wave * Sh::XI + q) % Sh::NXI;
    const int rr = n * Sh::RPI + (lane >> 4);
    const int node = j0 + rr < T ? j0 + rr : j0;
    xsrc[q] = X + static_cast<size_t>(node) * hid + 8 * ((lane & 15) ^ (rr & 15));
    xoff[q] = n * Sh::RPI * kL3RowBytes;
  }

  u32x4 wbuf[S][WT][4];
  // issue stage `stage` (clamped by the caller) into ring slot k
  auto load = [&](u32x4 (&w)[WT][4], uint8_t* xslot, int stage) {
    int ks = stage + rot;
    ks = ks >= nch ? ks - nch : ks;
    const int koff = ks * kL3Bk;
#pragma unroll
    for (int q = 0; q < Sh::XI; ++q) lds_dma16(xsrc[q] + koff, xslot + xoff[q]);
#pragma unroll
    for (int t = 0; t < WT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        w[t][i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wsrc[t][i] + koff));
  };

  f32x4 acc[WT][NT];
#pragma unroll
  for (int t = 0; t < WT; ++t)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[t][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint8_t* tp = tpose + wave * WT * kL3TileBytes;
  // each X fragment read from LDS feeds the WT tiles' products
  auto compute = [&](const u32x4 (&w)[WT][4], const uint8_t* xs) {
#pragma unroll
    for (int t = 0; t < WT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * i + lg;
        *reinterpret_cast<u32x4*>(tp + t * kL3TileBytes + r * kL3RowBytes + ((lr ^ r) << 4)) = w[t][i];
      }
    asm volatile("" ::: "memory");   // the tile's stores precede its reads
    // operand fragments of k-step s (32 k): A from the wave's tiles, B from
    // the X stage; the next step's fragments are read while this step's
    // products run, so the LDS latency hides behind the MFMAs
    bf16x8 fa[2][WT], fb[2][NT];
    auto fetch = [&](int s, int buf) {
      const int ch = 4 * s + lg;
#pragma unroll
      for (int t = 0; t < WT; ++t)
        fa[buf][t] = as_bf16x8(*reinterpret_cast<const u32x4*>(tp + t * kL3TileBytes + lr * kL3RowBytes +
                                                              ((ch ^ lr) << 4)));
#pragma unroll
      for (int n = 0; n < NT; ++n)
        fb[buf][n] = as_bf16x8(*reinterpret_cast<const u32x4*>(xs + (n * 16 + lr) * kL3RowBytes +
                                                              ((ch ^ lr) << 4)));
    };
    fetch(0, 0);
#pragma unroll
    for (int s = 0; s < kL3Bk / 32; ++s) {
      if (s + 1 < kL3Bk / 32) fetch(s + 1, (s + 1) & 1);
      // keep the scheduler from sinking the reads back to their uses
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int t = 0; t < WT; ++t)
          acc[t][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[s & 1][t], fb[s & 1][n], acc[t][n], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    asm volatile("" ::: "memory");   // and the next stage's stores follow them
  };

  load(wbuf[0], xring[0], 0);
  if constexpr (S > 2) load(wbuf[1], xring[1], 1 < nch ? 1 : nch - 1);
  if constexpr (S > 3) load(wbuf[2], xring[2], 2 < nch ? 2 : nch - 1);
  // one round = S pipeline steps; stage c + k is multiplied in step k
  auto round = [&](int c) {
#pragma unroll
    for (int k = 0; k < S; ++k) {
      const int cc = c + k;
      // this wave's loads of stage cc (its X share first, then its W
      // registers) are done once only the S-2 later stages remain in flight;
      // its LDS reads of stage cc-1 are done too (lgkmcnt(0))
      wait_vmcnt<(S - 2) * (Sh::XI + 4 * WT)>();
      stage_barrier();                       // every wave's X share of stage cc has landed
      const int nx = cc + S - 1 < nch ? cc + S - 1 : nch - 1;
      load(wbuf[(k + S - 1) % S], xring[(k + S - 1) % S], nx);
      // unconditional (nch % S == 0, and a wave without rows multiplies
      // in-bounds data it never stores): one straight-line path per step
      // keeps the compiler's load bookkeeping exact
      compute(wbuf[k], xring[k]);
    }
  };
  if constexpr (NCH > 0) {
#pragma unroll
    for (int c = 0; c < NCH; c += S) round(c);
  } else {
    for (int c = 0; c < nch; c += S) round(c);
  }
  wait_vmcnt<0>();   // no copy may land in LDS after the workgroup is gone

  const bool vec_ok = (V & 3) == 0;
  int vt[WT];   // first of the lane's four rows in tile t
#pragma unroll
  for (int t = 0; t < WT; ++t) vt[t] = tile0[t] + 4 * lg;
  if (logits) {   // the statistics path may run without materialised logits
#pragma unroll
    for (int t = 0; t < WT; ++t) {
      if (!live[t]) continue;
      const int v = vt[t];
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
  if constexpr (STATS) {
    // per node column: wave partial over the wave's rows, then the four
    // waves in LDS, then one partial per (node, workgroup).  The wave
    // partials live in the wave's own transposition tile, which its last
    // multiply has finished reading (LDS operations of a wave stay in
    // order), so the epilogue adds no LDS and the occupancy is unchanged.
    static_assert(Sh::TP * sizeof(StatPart) <= kL3TileBytes, "wave partials fit in a tile");
    StatPart* const wpart_own = reinterpret_cast<StatPart*>(tp);
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      StatPart p{-INFINITY, 0.f, 0.f, 0x7fffffff};
#pragma unroll
      for (int t = 0; t < WT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (live[t] && vt[t] + r < r1) take_max(p.zmax, p.idx, acc[t][n][r], vt[t] + r);
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1)
        take_max(p.zmax, p.idx, __shfl_xor(p.zmax, off, 64), __shfl_xor(p.idx, off, 64));
      if (p.zmax != -INFINITY) {
        const float my = p.zmax * inv_temp;
#pragma unroll
        for (int t = 0; t < WT; ++t)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if (live[t] && vt[t] + r < r1) {
              const float y = acc[t][n][r] * inv_temp - my;
              const float e = expf(y);
              p.Z += e;
              if (e > 0.f) p.S += y * e;
            }
          }
      }
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        p.Z += __shfl_xor(p.Z, off, 64);
        p.S += __shfl_xor(p.S, off, 64);
      }
      if (lg == 0) wpart_own[n * 16 + lr] = p;
    }
    __syncthreads();
    const int c = threadIdx.x;
    if (c < Sh::TP && j0 + c < T) {
      const StatPart* wpart = reinterpret_cast<const StatPart*>(tpose);
      constexpr int kStride = WT * kL3TileBytes / static_cast<int>(sizeof(StatPart));
      StatPart acc_p = wpart[c];
#pragma unroll
      for (int w = 1; w < kHybWaves; ++w) part_merge(acc_p, wpart[w * kStride + c], inv_temp);
      if (pcol >= 0) {
        // one partial per workgroup (column pcol of rows pstride long): a
        // workgroup's later slices fold into the partial of its first, which
        // this thread wrote itself
        StatPart* dst = part + static_cast<size_t>(j0 + c) * pstride + pcol;
        if (merge_prev) {
          StatPart prev = *dst;
          part_merge(prev, acc_p, inv_temp);
          acc_p = prev;
        }
        *dst = acc_p;
      } else {
        // the workgroup's slices: the combined partial in the first, neutral
        // partials in the others
        part[static_cast<size_t>(j0 + c) * G + WT * sl] = acc_p;
#pragma unroll
        for (int u = 1; u < WT; ++u)
          part[static_cast<size_t>(j0 + c) * G + WT * sl + u] = StatPart{-INFINITY, 0.f, 0.f, 0x7fffffff};
      }
    }
  }
}

template <int NT, int S, int NCH, bool STATS, int WT = 1>
__global__ __launch_bounds__(kHybThreads) void lm_head_hyb_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    int T, int hid, int V, int G, float inv_temp, StatPart* __restrict__ part) {
  constexpr int XSTAGE = HybShape<NT>::TP * kL3RowBytes;   // bytes of one X stage
  __shared__ __attribute__((aligned(16))) uint8_t xslot0[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot1[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot2[S > 2 ? XSTAGE : 16];
  __shared__ __attribute__((aligned(16))) uint8_t xslot3[S > 3 ? XSTAGE : 16];
  __shared__ __attribute__((aligned(16))) uint8_t tpose[kHybWaves * WT * kL3TileBytes];
  // 1-D grid over (slice group, pass, XCD): the passes of one slice share an
  // XCD (dispatch is round-robin over 8 XCDs) and start together, so a W
  // stage fetched from HBM by one of them is an L2 hit for the others
  const int passes = (T + HybShape<NT>::TP - 1) / HybShape<NT>::TP;
  const int bid = blockIdx.x, r = bid >> 3;
  const int pass = r % passes, slice = (r / passes) * 8 + (bid & 7);
  if (slice >= G / WT) return;
  hyb_body<NT, S, NCH, STATS, WT>(xslot0, xslot1, xslot2, xslot3, tpose, X, W, logits, T, hid, V,
                                  G, inv_temp, part, pass * HybShape<NT>::TP, slice);
}

// Trees of up to 32 nodes inside a step: one workgroup per pair of
// consecutive vocabulary slices ((G + 1) / 2 workgroups: one per CU at the
// 7B vocabulary, which leaves room beside it for the step's attention).
// Each wave streams two 16-row W tiles, so the pipeline runs unbroken over
// both slices (taking the two slices one after the other drains and refills
// it in between: 49.0 against 46.8 us for the 27-node tree at 7B shapes)
// and every X fragment read from LDS feeds two products.  One statistics
// partial per workgroup and node: column = pair index, rows (G + 1) / 2
// long, the layout the step's finalize merges in one pass.
template <int NT, int NCH>
__global__ __launch_bounds__(kHybThreads) void lm_head_pair_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    int T, int hid, int V, int G, float inv_temp, StatPart* __restrict__ part) {
  constexpr int XSTAGE = HybShape<NT>::TP * kL3RowBytes;
  __shared__ __attribute__((aligned(16))) uint8_t xslot0[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot1[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot2[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot3[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t tpose[kHybWaves * 2 * kL3TileBytes];
  hyb_body<NT, 4, NCH, true, 2>(xslot0, xslot1, xslot2, xslot3, tpose, X, W, logits, T, hid, V, G,
                                inv_temp, part, 0, blockIdx.x, blockIdx.x, gridDim.x, false);
}

// The same kernel with the node count read from device memory (*T_dev), for
// steps whose tree is chosen on the GPU.  Two kernels share the range so that
// each keeps the LDS of its own node tile (and with it room on the CUs for
// the attention running alongside): the small one takes trees of up to 32
// nodes (16- or 32-node tile), the large one trees of 33..128 nodes (one
// 128-node pass); each leaves at once when the tree is not in its range.
// Statistics partials only.
template <int NCH>
__global__ __launch_bounds__(kHybThreads) void lm_head_dyn_small_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    const int* __restrict__ T_dev, int hid, int V, int G, float inv_temp,
    StatPart* __restrict__ part) {
  constexpr int XSTAGE = HybShape<2>::TP * kL3RowBytes;
  __shared__ __attribute__((aligned(16))) uint8_t xslot0[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot1[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot2[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot3[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t tpose[kHybWaves * 2 * kL3TileBytes];
  const int T = __builtin_amdgcn_readfirstlane(*T_dev);
  if (T > kStepSmallT) return;
  // a pair of vocabulary slices per workgroup (the grid is half the
  // slices), as the host-sized pair kernel, with its partial layout
  if (T <= 16)
    hyb_body<1, 4, NCH, true, 2>(xslot0, xslot1, xslot2, xslot3, tpose, X, W, logits, T, hid, V, G,
                                 inv_temp, part, 0, blockIdx.x, blockIdx.x, gridDim.x, false);
  else
    hyb_body<2, 4, NCH, true, 2>(xslot0, xslot1, xslot2, xslot3, tpose, X, W, logits, T, hid, V, G,
                                 inv_temp, part, 0, blockIdx.x, blockIdx.x, gridDim.x, false);
}

template <int NCH, int WT>
__global__ __launch_bounds__(kHybThreads) void lm_head_dyn_large_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    const int* __restrict__ T_dev, int hid, int V, int G, float inv_temp,
    StatPart* __restrict__ part) {
  constexpr int XSTAGE = HybShape<8>::TP * kL3RowBytes;
  __shared__ __attribute__((aligned(16))) uint8_t xslot0[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t xslot1[XSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t tpose[kHybWaves * WT * kL3TileBytes];
  const int T = __builtin_amdgcn_readfirstlane(*T_dev);
  if (T > kStepSmallT)
    hyb_body<8, 2, NCH, true, WT>(xslot0, xslot1, xslot0, xslot1, tpose, X, W, logits, T, hid, V,
                                  G, inv_temp, part, 0, blockIdx.x);
}

// Largest vocabulary slice slice_begin() produces for G workgroups (host copy
// of the same arithmetic).
int max_slice(int V, int G) {
  auto begin = [&](int b) {
    return b >= G ? V : static_cast<int>((static_cast<long long>(V) * b / G) & ~3ll);
  };
  int m = 0;
  for (int b = 0; b < G; ++b) m = std::max(m, begin(b + 1) - begin(b));
  return m;
}

// Compute units of the current device (queried once per device).
int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// Combines the G partials of each node into its statistics: one wavefront
// per node, kFinNodes nodes per workgroup.
constexpr int kFinNodes = 4;
__global__ __launch_bounds__(64 * kFinNodes) void stats_finalize_kernel(
    const StatPart* __restrict__ part, int G, int T, float inv_temp, float* __restrict__ entropy,
    float* __restrict__ top1p, int* __restrict__ argmax) {
  const int node = blockIdx.x * kFinNodes + (threadIdx.x >> 6);
  if (node >= T) return;   // whole wavefronts
  // up to 2048 partials per row (a 128256-entry vocabulary writes 2004) in
  // registers, 32 per lane, so the row's loads go out together
  const int rows[1] = {node};
  StatPart o[1];
  if (G <= 64 * kMergeRegParts)
    merge_rows<1>(part, rows, G, inv_temp, o);
  else
    merge_rows<1, 4 * kMergeRegParts>(part, rows, G, inv_temp, o);
  const StatPart& a = o[0];
  if ((threadIdx.x & 63) == 0) {
    if (entropy) entropy[node] = part_entropy(a);
    if (top1p) top1p[node] = part_top1p(a);
    if (argmax) argmax[node] = a.idx;
  }
}

// Workgroups of the streaming LM-head grid: slices of at most 64 rows, and a
// whole multiple of the CU count, so that every CU streams the same number
// of bytes (a partial extra round of workgroups on a few CUs costs ~20% at
// 7B shapes).
int hyb_grid_uncached(int V, int cus) {
  constexpr int rows = 16 * kHybWaves;
  const int max_g = (V + 3) / 4;
  int G = cus;
  while (G < max_g && max_slice(V, G) > rows) G += cus;
  return G < max_g ? G : max_g;
}

// (The search above walks every slice; a call in the step's critical path
// takes the last answer for the same CU count and vocabulary instead.)
int hyb_grid(int V) {
  thread_local int last_cus = -1, last_V = -1, last_G = 0;
  const int cus = device_cus();
  if (cus != last_cus || V != last_V) {
    last_G = hyb_grid_uncached(V, cus);
    last_cus = cus;
    last_V = V;
  }
  return last_G;
}

// ev0 / ev1 (may be NULL) are recorded on the stream right before and after
// the launch.
// WT = 2 pairs consecutive slices in one workgroup (G / 2 workgroups; the
// caller keeps that at least one per CU).
template <int NT, int S, int NCH, bool STATS = false, int WT = 1>
int32_t launch_lm_hyb(const uint16_t* X, const uint16_t* W, float* logits, int T, int hid, int V,
                      hipStream_t s, float inv_temp = 1.f, StatPart* part = nullptr,
                      hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr) {
  const int G = hyb_grid(V);
  const int passes = (T + NT * 16 - 1) / (NT * 16);
  const int groups = (G / WT + 7) / 8;   // slices in groups of 8, one per XCD
  if (ev0)
    if (int32_t rc = hip_status(hipEventRecord(ev0, s), "hipEventRecord")) return rc;
  hipLaunchKernelGGL((lm_head_hyb_kernel<NT, S, NCH, STATS, WT>), dim3(groups * passes * 8),
                     dim3(kHybThreads), 0, s, X, W, logits, T, hid, V, G, inv_temp, part);
  if (int32_t rc = launch_status("verify_logits launch")) return rc;
  return ev1 ? hip_status(hipEventRecord(ev1, s), "hipEventRecord") : ENTMTP_OK;
}

// Streaming LM head with fused statistics partials, then the per-node
// finalize; false when the streaming kernel does not apply to hid.
// beside: other work (the step's attention) runs beside the LM head.
template <bool STATS>
bool launch_hyb_dispatch(const uint16_t* X, const uint16_t* W, float* logits, int T, int hid, int V,
                         hipStream_t s, float inv_temp, StatPart* part, int32_t* rc,
                         hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr, bool beside = false) {
  // large node tiles pair slices per workgroup (each X fragment read from
  // LDS then feeds two W tiles) when that still leaves a workgroup per CU;
  // 128-node tiles only beside other work: alone, two unpaired workgroups
  // per CU keep more of W in flight (the batch-8 LM head: 259 -> 247 us),
  // but they fill the CU's LDS, and beside the 13B step's attention they lost
  // (96 -> 106 us)
  // many rows: the tiled contraction reads W once per 128 rows with each
  // LDS byte feeding more products
  if (lm_gemm_takes(T, hid, hyb_grid(V), device_cus())) {
    if (ev0)
      if ((*rc = hip_status(hipEventRecord(ev0, s), "hipEventRecord"))) return true;
    *rc = launch_lm_gemm(reinterpret_cast<const entmtp_bf16*>(X),
                         reinterpret_cast<const entmtp_bf16*>(W), logits, T, hid, V, hyb_grid(V),
                         inv_temp, STATS ? part : nullptr, device_cus(), s);
    if (*rc == ENTMTP_OK && ev1) *rc = hip_status(hipEventRecord(ev1, s), "hipEventRecord");
    return true;
  }
  const bool pair = hyb_grid(V) >= 2 * device_cus();
  const bool pair128 = pair && beside;
  auto go = [&](auto nch) {
    constexpr int NCH = decltype(nch)::value;
    if (T <= 16)
      *rc = launch_lm_hyb<1, 4, NCH, STATS>(X, W, logits, T, hid, V, s, inv_temp, part, ev0, ev1);
    else if (T <= 32)
      *rc = launch_lm_hyb<2, 4, NCH, STATS>(X, W, logits, T, hid, V, s, inv_temp, part, ev0, ev1);
    else if (T <= 64)
      *rc = pair ? launch_lm_hyb<4, kHybS4, NCH, STATS, kHybW4>(X, W, logits, T, hid, V, s, inv_temp, part, ev0, ev1)
                 : launch_lm_hyb<4, 4, NCH, STATS>(X, W, logits, T, hid, V, s, inv_temp, part, ev0, ev1);
    else
      *rc = pair128 ? launch_lm_hyb<8, kHybS8, NCH, STATS, kHybW8>(X, W, logits, T, hid, V, s, inv_temp, part, ev0, ev1)
                    : launch_lm_hyb<8, 2, NCH, STATS>(X, W, logits, T, hid, V, s, inv_temp, part, ev0, ev1);
  };
  if (hid == 4096) {              // the 7B hidden size: K loop fully unrolled
    go(std::integral_constant<int, 32>{});
    return true;
  }
  if (hid == 5120) {              // the 13B hidden size
    go(std::integral_constant<int, 40>{});
    return true;
  }
  if (hid % (4 * kL3Bk) == 0) {   // a whole number of 4-stage rounds
    go(std::integral_constant<int, 0>{});
    return true;
  }
  return false;
}

template <int NT, int S>
int32_t launch_lm_lds(const uint16_t* X, const uint16_t* W, float* logits, int T, int hid, int V,
                      hipStream_t s) {
  constexpr int rows = 16 * kL3Waves;   // 128 rows per slice at most
  const int want = (V + rows - 5) / (rows - 4);
  int G = want > 256 ? want : 256;
  const int max_g = (V + 3) / 4;
  G = G < max_g ? G : max_g;
  const int passes = (T + NT * 16 - 1) / (NT * 16);
  hipLaunchKernelGGL((lm_head_lds_kernel<NT, S>), dim3(G, passes), dim3(kL3Threads), 0, s, X, W,
                     logits, T, hid, V, G);
  return launch_status("verify_logits launch");
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

int stats_slices(int V) { return hyb_grid(V); }

int step_small_parts(int V) { return (hyb_grid(V) + 1) / 2; }

int32_t launch_step_partials(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, int T, int hid,
                             int V, float inv_temp, float* logits, void* partials, int* n_parts,
                             hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  auto* part = static_cast<StatPart*>(partials);
  const auto* X = reinterpret_cast<const uint16_t*>(hidden);
  const auto* W = reinterpret_cast<const uint16_t*>(w_lm);
  *n_parts = step_small_parts(V);
  if (T > kStepSmallT) {   // the step's configuration was checked: hid is a multiple of 4 rounds
    *n_parts = hyb_grid(V);
    int32_t rc = ENTMTP_OK;
    if (!launch_hyb_dispatch<true>(X, W, logits, T, hid, V, s, inv_temp, part, &rc, ev0, ev1, true))
      return fail(ENTMTP_EINVAL, "hid = %d: no streaming LM head", hid);
    return rc;
  }
  const int G = hyb_grid(V);
  const dim3 grid((G + 1) / 2);
  if (ev0)
    if (int32_t rc = hip_status(hipEventRecord(ev0, s), "hipEventRecord")) return rc;
  auto go = [&](auto k) {
    hipLaunchKernelGGL(k, grid, dim3(kHybThreads), 0, s, X, W, logits, T, hid, V, G, inv_temp, part);
  };
  if (hid == 32 * kL3Bk) {
    if (T <= 16) go(lm_head_pair_kernel<1, 32>); else go(lm_head_pair_kernel<2, 32>);
  } else if (hid == 40 * kL3Bk) {
    if (T <= 16) go(lm_head_pair_kernel<1, 40>); else go(lm_head_pair_kernel<2, 40>);
  } else {
    if (T <= 16) go(lm_head_pair_kernel<1, 0>); else go(lm_head_pair_kernel<2, 0>);
  }
  if (int32_t rc = launch_status("verify_logits (step) launch")) return rc;
  return ev1 ? hip_status(hipEventRecord(ev1, s), "hipEventRecord") : ENTMTP_OK;
}

int32_t launch_partials_device_T(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                 const int* T_dev, int T_max, int hid, int V, float inv_temp,
                                 void* partials, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (T_max < 1 || T_max > 128 || hid % (4 * kL3Bk))
    return fail(ENTMTP_EINVAL, "device-sized LM head: T_max %d (at most 128), hid %d (multiple of %d)",
                T_max, hid, 4 * kL3Bk);
  const int G = hyb_grid(V);
  auto* part = static_cast<StatPart*>(partials);
  const auto* X = reinterpret_cast<const uint16_t*>(hidden);
  const auto* W = reinterpret_cast<const uint16_t*>(w_lm);
  // the large kernel pairs slices per workgroup (as the host-sized one) when
  // that leaves a workgroup per CU: half the workgroups to place when it has
  // nothing to do
  const int large_wt = G >= 2 * device_cus() ? 2 : 1;
  auto both = [&](auto small, auto large) -> int32_t {
    if (ev0)
      if (int32_t rc = hip_status(hipEventRecord(ev0, s), "hipEventRecord")) return rc;
    hipLaunchKernelGGL(small, dim3((G + 1) / 2), dim3(kHybThreads), 0, s, X, W, nullptr, T_dev,
                       hid, V, G, inv_temp, part);
    if (int32_t rc = launch_status("verify_logits (device-sized, small) launch")) return rc;
    if (T_max > 32) {   // some bank tree needs the large kernel
      hipLaunchKernelGGL(large, dim3(G / large_wt), dim3(kHybThreads), 0, s, X, W, nullptr, T_dev,
                         hid, V, G, inv_temp, part);
      if (int32_t rc = launch_status("verify_logits (device-sized, large) launch")) return rc;
    }
    return ev1 ? hip_status(hipEventRecord(ev1, s), "hipEventRecord") : ENTMTP_OK;
  };
  if (hid == 32 * kL3Bk)
    return large_wt == 2 ? both(lm_head_dyn_small_kernel<32>, lm_head_dyn_large_kernel<32, 2>)
                         : both(lm_head_dyn_small_kernel<32>, lm_head_dyn_large_kernel<32, 1>);
  if (hid == 40 * kL3Bk)
    return large_wt == 2 ? both(lm_head_dyn_small_kernel<40>, lm_head_dyn_large_kernel<40, 2>)
                         : both(lm_head_dyn_small_kernel<40>, lm_head_dyn_large_kernel<40, 1>);
  return large_wt == 2 ? both(lm_head_dyn_small_kernel<0>, lm_head_dyn_large_kernel<0, 2>)
                       : both(lm_head_dyn_small_kernel<0>, lm_head_dyn_large_kernel<0, 1>);
}

int32_t launch_stats_finalize(const void* partials, int T, int V, float inv_temp, float* entropy,
                              float* top1p, int* argmax, hipStream_t s) {
  hipLaunchKernelGGL(stats_finalize_kernel, dim3((T + kFinNodes - 1) / kFinNodes),
                     dim3(64 * kFinNodes), 0, s, static_cast<const StatPart*>(partials),
                     hyb_grid(V), T, inv_temp, entropy, top1p, argmax);
  return launch_status("stats_finalize launch");
}

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
  int32_t rc = ENTMTP_OK;
  if (launch_hyb_dispatch<false>(hidden, w_lm, logits, T, hid, V, s, 1.f, nullptr, &rc)) return rc;
  if (hid % kL3Bk == 0) {
    if (T <= 16) return launch_lm_lds<1, 4>(hidden, w_lm, logits, T, hid, V, s);
    if (T <= 32) return launch_lm_lds<2, 4>(hidden, w_lm, logits, T, hid, V, s);
    if (T <= 64) return launch_lm_lds<4, 3>(hidden, w_lm, logits, T, hid, V, s);
    return launch_lm_lds<8, 2>(hidden, w_lm, logits, T, hid, V, s);
  }
  if (T <= 16) return launch_lm<1, 256>(hidden, w_lm, logits, T, hid, V, s);
  if (T <= 32) return launch_lm<2, 256>(hidden, w_lm, logits, T, hid, V, s);
  if (T <= 64) return launch_lm<4, 128>(hidden, w_lm, logits, T, hid, V, s);
  return launch_lm<8, 128>(hidden, w_lm, logits, T, hid, V, s);
}

extern "C" size_t entmtp_stats_partials_bytes(int32_t T, int32_t hid, int32_t V) {
  if (T < 1 || T > 4096 || V < 1 || hid < 8 || hid % (4 * kL3Bk)) return 0;
  return static_cast<size_t>(T) * hyb_grid(V) * sizeof(StatPart);
}

extern "C" int32_t entmtp_verify_logits_partials(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                                 int32_t T, int32_t hid, int32_t V, float inv_temp,
                                                 float* logits, void* partials,
                                                 size_t partials_bytes, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(hidden && w_lm && partials, ENTMTP_EINVAL,
                   "hidden, w_lm and partials must be non-NULL");
  ENTMTP_CHECK_ARG(T >= 1 && T <= 4096, ENTMTP_EINVAL, "T = %d outside [1, 4096]", T);
  ENTMTP_CHECK_ARG(hid >= 4 * kL3Bk && hid % (4 * kL3Bk) == 0, ENTMTP_EINVAL,
                   "hid = %d: the fused path needs a multiple of %d", hid, 4 * kL3Bk);
  ENTMTP_CHECK_ARG(V >= 1, ENTMTP_EINVAL, "V = %d < 1", V);
  ENTMTP_CHECK_ARG(inv_temp > 0.f && inv_temp < INFINITY, ENTMTP_EINVAL,
                   "inv_temp = %g must be positive and finite", static_cast<double>(inv_temp));
  ENTMTP_CHECK_ARG(aligned16(hidden) && aligned16(w_lm) && aligned16(logits) && aligned16(partials),
                   ENTMTP_EINVAL, "hidden, w_lm, logits and partials must be 16-byte aligned");
  const size_t need = entmtp_stats_partials_bytes(T, hid, V);
  ENTMTP_CHECK_ARG(partials_bytes >= need, ENTMTP_ENOSPC, "partials buffer has %zu bytes, needs %zu",
                   partials_bytes, need);
  int32_t rc = ENTMTP_OK;
  launch_hyb_dispatch<true>(hidden, w_lm, logits, T, hid, V, static_cast<hipStream_t>(stream),
                            inv_temp, static_cast<StatPart*>(partials), &rc);
  return rc;
}

extern "C" int32_t entmtp_stats_finalize(const void* partials, int32_t T, int32_t V, float inv_temp,
                                         float* entropy, float* top1p, int32_t* argmax,
                                         void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(partials != nullptr, ENTMTP_EINVAL, "partials is NULL");
  ENTMTP_CHECK_ARG(T >= 1 && T <= 4096 && V >= 1, ENTMTP_EINVAL, "T = %d, V = %d out of range", T, V);
  ENTMTP_CHECK_ARG(inv_temp > 0.f && inv_temp < INFINITY, ENTMTP_EINVAL,
                   "inv_temp = %g must be positive and finite", static_cast<double>(inv_temp));
  if (!entropy && !top1p && !argmax) return ENTMTP_OK;
  return launch_stats_finalize(partials, T, V, inv_temp, entropy, top1p, argmax,
                               static_cast<hipStream_t>(stream));
}

extern "C" size_t entmtp_verify_logits_stats_workspace(int32_t T, int32_t hid, int32_t V) {
  if (T < 1 || T > 4096 || V < 1 || hid < 8 || hid % 8) return 0;
  const size_t p = entmtp_stats_partials_bytes(T, hid, V);
  return p ? p : 256;   // other hidden sizes: separate kernels, no partials
}

extern "C" int32_t entmtp_verify_logits_stats(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                              int32_t T, int32_t hid, int32_t V, float inv_temp,
                                              float* logits, float* entropy, float* top1p,
                                              int32_t* argmax, void* workspace,
                                              size_t workspace_bytes, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(hid >= 8 && hid % 8 == 0, ENTMTP_EINVAL, "hid = %d must be a positive multiple of 8", hid);
  if (entmtp_stats_partials_bytes(T, hid, V) > 0) {
    if (int32_t rc = entmtp_verify_logits_partials(hidden, w_lm, T, hid, V, inv_temp, logits,
                                                   workspace, workspace_bytes, stream))
      return rc;
    return entmtp_stats_finalize(workspace, T, V, inv_temp, entropy, top1p, argmax, stream);
  }
  // other hidden sizes: logits first, then the statistics pass over them
  if (int32_t rc = entmtp_verify_logits(hidden, w_lm, T, hid, V, logits, stream)) return rc;
  return entmtp_logit_stats(logits, T, V, inv_temp, entropy, top1p, argmax, stream);
}
