// Tree-masked attention of the verification pass.
//
// §2.3: the draft tree is verified in a single sparse forward pass of the
// target model with a precomputed tree attention mask and position offsets;
// §3.2 names the mask size among the per-step verifier costs.  Node i of the
// tree attends to the whole prefix and to the nodes on its own root-to-node
// path; it sits at sequence position prefix_len + depth(i).
//
// Two kernels, both on the caller's stream:
//  1. attend: flash-decoding over the cache, one of two kernels.  The
//     queries and the tree's keys are rotated to their positions as they are
//     loaded (fp64 angles from a per-workgroup LDS table over the tree's
//     depths, one bf16 rounding); the tree's keys and values come from the
//     step's inputs rather than the cache, and the workgroups of the first
//     query group write them (keys rotated) into cache slots [L, L+T) for
//     the steps after this one.
//     Trees of up to 32 query rows per KV head: a workgroup owns one (KV
//     head, 32-query tile, key split); its four waves take interleaved 32-key
//     blocks, each wave loading its next block while it multiplies the
//     current one (K two blocks deep in registers, V one); the tile's
//     fragments live once per workgroup in LDS, and the four waves merge in
//     LDS at the end.  Larger trees: a workgroup owns four tiles, one per
//     wave, and the waves walk the same key blocks, staged once per
//     workgroup in LDS (K as rows, V transposed), so a block is read once per
//     128 rows; that kernel stays under 256 registers per lane, two
//     workgroups per CU.
//     S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_32x32x16_bf16, V
//     transposed through LDS, P never leaving registers (the S^T accumulator
//     layout is re-read as the B operand of the PV product after a fixed key
//     permutation).  Blocks wholly inside the prefix skip the mask; the
//     others take a 32-bit window cut from the node's ancestor bitmask.
//     Online softmax in fp32, base 2, with a lazily raised running max (the
//     accumulators are rescaled only when a block's max passes the reference
//     by more than 2^8).
//  2. merge: combines the splits' partials: (max, sum) in fp32 and the
//     output normalised by its sum, in bf16 (half the bytes of fp32; a
//     normalised partial stays within the range of the values).
//     Skipped when a single split covers the keys.
#include <cfloat>
#include <cmath>
#include <mutex>

#include "common.hpp"

namespace entmtp {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int HD = ENTMTP_HEAD_DIM;  // 128
constexpr int kAttnThreads = 256;
constexpr int kAttnWaves = 4;
constexpr int KB = 32;               // keys per block
constexpr int kQTile = 32;           // query rows per tile
constexpr float kLazyLog2 = 8.f;     // the running max is raised only past this many doublings
constexpr int VT_LD = 36;            // bf16 per V^T row in LDS (32 keys + pad)
constexpr int kMaxSplits = 32;
constexpr int kMinBlocksPerSplit = 4;   // one block per wave at least
// A batch's blocks-per-split target: its key-block streams (one per KV head,
// query group and 32-key block: what a workgroup reads) over this many
// workgroups per CU.
constexpr int kBatchWgPerCu = 3;
constexpr int kMaxSeqs = ENTMTP_B_MAX;

__host__ __device__ inline int rows_padded(int G, int T) {
  return (G * T + kQTile - 1) / kQTile * kQTile;
}

// Workgroups along the query rows: groups of nt 32-row tiles.
__host__ __device__ inline int query_groups(int nqt, int nt) { return (nqt + nt - 1) / nt; }

// Query tiles per workgroup for a tree: one up to one tile of rows per KV
// head, four (one per wave) above.  (The two-tile form -- both tiles in every
// wave -- measured slower than four tiles with two waves idle: 23.5 against
// 19.8 us at 64 rows and prefix 4096.)
__host__ __device__ inline int tree_tiles(int G, int T) { return G * T > kQTile ? 4 : 1; }

__host__ __device__ inline int split_bound(int nblocks) {
  int b = nblocks / kMinBlocksPerSplit;
  b = b < 1 ? 1 : b;
  return b > kMaxSplits ? kMaxSplits : b;
}

// Split count of a lone sequence: one workgroup fits per CU, so pick the
// count that fills the CUs in whole rounds -- the first (1..bound) whose last
// round is at least 90% full, else the fullest one seen (integer arithmetic,
// so that the host and the device choose alike).
__host__ __device__ inline int split_for_bound(int bound, int base_wg, int cus) {
  int best = 1;
  long long best_wg = 0, best_rounds = 1;
  for (int ns = 1; ns <= bound; ++ns) {
    const long long wg = static_cast<long long>(base_wg) * ns;
    const long long rounds = (wg + cus - 1) / cus;
    if (wg * best_rounds > best_wg * rounds) {   // fill wg / (rounds * cus) improves
      best_wg = wg;
      best_rounds = rounds;
      best = ns;
    }
    if (10 * wg >= 9 * rounds * cus) break;
  }
  return best;
}

// Workgroups of an instance resident per CU: two for the four-tile kernel
// (under 256 registers per lane), one for the others.
__host__ __device__ inline int wg_per_cu(int nt) { return nt == 4 ? 2 : 1; }

__host__ __device__ inline int split_single(int nblocks, int base_wg, int cus) {
  return split_for_bound(split_bound(nblocks), base_wg, cus);
}

// ----------------------------------------------------------- descriptors --

// One sequence of a (possibly batched) call, planned on the host.
struct SeqPlan {
  uint16_t* kc;            // [Hkv][cap][HD] this sequence's cache
  uint16_t* vc;
  const uint32_t* mask;    // [T][ENTMTP_MASK_WORDS] its tree's ancestor bitmask
  const int* depth;        // [T]
  int T, L, row0;          // nodes, prefix length, first row in the concatenated q / out
  int D;                   // depth of the tree's deepest node
  int rows_pad, nqt, nqg, nsplit, bps;   // padded rows, query tiles, query groups, splits
  int nt;                  // query tiles per workgroup the call's plan gives it
  int item0;               // first attend workgroup of the sequence
  int merge0;              // first merge block of the sequence
  long long part_off;      // row offset of its split partials
};

// A bank tree as a device-planned batch finds it (kernel arguments).
struct TreeHdr {
  int T, D, off_mask, off_depth;
};
constexpr int kMaxTreesArg = 32;   // bank trees a device-planned batch can name

struct BatchArgs {
  SeqPlan s[kMaxSeqs];
  // device-planned batch: sequence b's tree, prefix length and first row
  // come from device arrays (topo_dev[b], len_dev[b], row_off_dev[b]); the
  // host fixed its caches and its grid, merge and partial ranges (at strides
  // sized for the bank's largest plan), and every workgroup derives the
  // plan the host would have made (plan_call) from those arrays
  const int32_t* topo_dev;
  const int32_t* len_dev;
  const int32_t* row_off_dev;   // [B + 1]
  int rows_cap;                 // rows q / k_tree / v_tree / out hold
  int n_trees;
  TreeHdr trees[kMaxTreesArg];
  // device-planned single sequence (a tree chosen on the GPU): when dev is
  // set, sequence 0's tree, prefix length and split plan come from *dev, the
  // bank descriptors and the CU count, and the grids are sized for the
  // largest plan
  const DevStep* dev;
  const DevTopo* topos;
  const uint8_t* arena;
  int cus;
  int nt;                  // query tiles per workgroup of the launched kernel (1 or 2)
  int B, G, Hq, Hkv, cap;
  float scale_log2;
  double theta;            // rotation base (0: no rotation)
  double freq[HD / 2];     // theta^(-2c/d) of pair c, computed on the host
  const uint16_t* q;       // [rows][Hq][HD] (rows = sum of T, sequence after sequence)
  const uint16_t* kt;      // [rows][Hkv][HD]
  const uint16_t* vt;
  uint16_t* part_o;        // [part rows][HD] bf16: the split's output, normalised by its sum
  float* part_ml;          // [part rows][2]
  uint16_t* out;           // [rows][Hq][HD]
};
static_assert(sizeof(BatchArgs) <= 4096, "kernel arguments are limited to 4 KB");

// Sequence that owns index `x` of a grid whose per-sequence ranges start at
// `first(b)` (uniform per workgroup; at most kMaxSeqs steps).
template <typename F>
__device__ __forceinline__ int seq_of(const BatchArgs& p, int x, F first) {
  int b = 0;
  while (b + 1 < p.B && x >= first(p.s[b + 1])) ++b;
  return b;
}

// Plan of sequence b: the host's, or -- for a device-planned call -- the
// plan the host would make for the tree and prefix length the device holds
// (same arithmetic), with the caches the host passed.
__device__ __forceinline__ SeqPlan resolve(const BatchArgs& p, int b) {
  if (!p.dev) return p.s[b];
  SeqPlan q = p.s[0];
  const DevStep st = *p.dev;
  const DevTopo* t = p.topos + st.rung;   // read in place (no local copy to index)
  q.T = st.T;
  q.L = st.L;
  q.D = t->D;
  if (q.L < 0 || q.T < 1 || q.L + q.T > p.cap) {   // outside the cache: no attention at all
    q.T = 0;
    q.L = 0;
    q.nsplit = 1;
    q.nqt = 0;
    q.nqg = 0;
    return q;
  }
  q.mask = reinterpret_cast<const uint32_t*>(p.arena + t->off_mask);
  q.depth = reinterpret_cast<const int*>(p.arena + t->off_depth);
  q.row0 = 0;
  q.rows_pad = rows_padded(p.G, q.T);
  q.nqt = q.rows_pad / kQTile;
  q.nqg = query_groups(q.nqt, tree_tiles(p.G, q.T));
  const int nblocks = (q.L + q.T + KB - 1) / KB;
  const int ns = t->splits[split_bound(nblocks)];   // = split_single(nblocks, Hkv * nqg, cus * wg_per_cu)
  q.bps = (nblocks + ns - 1) / ns;
  q.nsplit = (nblocks + q.bps - 1) / q.bps;
  q.item0 = 0;
  q.merge0 = 0;
  q.part_off = 0;
  return q;
}

// Plan of sequence b of a device-planned batch.  Lane i of each wavefront
// reads sequence i's entries; a sequence whose tree index lies outside the
// bank, whose prefix length is negative or leaves no room for its tree in
// the cache, or whose tree rows [row_off[b], row_off[b] + T) do not lie in
// [row_off[b], row_off[b + 1]) and the row capacity has no work (T = 0) and
// counts for nothing in the batch plan.
// The rest is plan_call's arithmetic: the batch's tile count is the largest
// any sequence needs, and a batch of several shares one blocks-per-split
// target.  Called by whole wavefronts.
__device__ __forceinline__ SeqPlan resolve_batch(const BatchArgs& p, int b) {
  SeqPlan q = p.s[b];   // caches and the fixed ranges
  const int lane = threadIdx.x & 63;
  int tr = -1, L = -1, r0 = -1, r1 = -1;
  if (lane < p.B) {
    tr = p.topo_dev[lane];
    L = p.len_dev[lane];
    r0 = p.row_off_dev[lane];
    r1 = p.row_off_dev[lane + 1];
  }
  // every bank tree's size, lane k holding tree k's (requested with the
  // entries above, so one memory round trip covers both)
  const int tree_T = lane < p.n_trees ? p.trees[lane].T : 0;
  const bool named = lane < p.B && tr >= 0 && tr < p.n_trees;
  const int T_named = __shfl(tree_T, named ? tr : 0, 64);
  int T = named ? T_named : 0;
  const long long end = static_cast<long long>(r0) + T;   // (64-bit: the entries are unchecked)
  const bool ok = named && L >= 0 && static_cast<long long>(L) + T <= p.cap && r0 >= 0 &&
                  end <= r1 && end <= p.rows_cap;
  if (!ok) T = 0;
  const int nblocks = T ? (L + T + KB - 1) / KB : 0;
  int nt = T ? tree_tiles(p.G, T) : 1;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) nt = max(nt, __shfl_xor(nt, off, 64));
  long long work =
      T ? static_cast<long long>(p.Hkv) * query_groups(rows_padded(p.G, T) / kQTile, nt) * nblocks
        : 0;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) work += __shfl_xor(work, off, 64);
  const int Tb = __shfl(T, b, 64);
  if (Tb == 0) {
    q.T = 0;
    q.L = 0;
    q.nsplit = 1;
    q.nqt = 0;
    q.nqg = 0;
    q.nt = nt;
    return q;
  }
  const int trb = __shfl(tr, b, 64);
  const TreeHdr& h = p.trees[trb];
  q.T = Tb;
  q.L = __shfl(L, b, 64);
  q.row0 = __shfl(r0, b, 64);
  q.D = h.D;
  q.mask = reinterpret_cast<const uint32_t*>(p.arena + h.off_mask);
  q.depth = reinterpret_cast<const int*>(p.arena + h.off_depth);
  q.nt = nt;
  q.rows_pad = rows_padded(p.G, q.T);
  q.nqt = q.rows_pad / kQTile;
  q.nqg = query_groups(q.nqt, nt);
  const int nb = (q.L + q.T + KB - 1) / KB;
  int ns;
  if (p.B == 1) {
    ns = split_single(nb, p.Hkv * q.nqg, p.cus * wg_per_cu(nt));
  } else {
    const long long per_wg = (work + kBatchWgPerCu * p.cus - 1) / (kBatchWgPerCu * p.cus);
    const int target_bps = static_cast<int>(per_wg > kMinBlocksPerSplit ? per_wg : kMinBlocksPerSplit);
    ns = (nb + target_bps - 1) / target_bps;
    const int bound = split_bound(nb);
    ns = ns < 1 ? 1 : (ns > bound ? bound : ns);
  }
  q.bps = (nb + ns - 1) / ns;
  q.nsplit = (nb + q.bps - 1) / q.bps;
  return q;
}

// ------------------------------------------------------------------ RoPE --

// Angles of a tree's positions: tab[d * 64 + c] = (cos, sin) of the turn of
// pair (c, c + 64) at position L + d, d = 0..D, in fp64 (pos * freq[c],
// freq[c] = theta^(-2c/d) from the host), followed by the same table in
// fp32 (for the queries), filled by the workgroup's threads (a multiple of
// 64: each keeps one pair's frequency).  The tables live in the kernel's
// dynamic LDS, sized by the host for the deepest tree of the launch.
constexpr int kRopePairs = HD / 2;
inline size_t rope_lds_bytes(int D, double theta) {
  return theta > 0.0 ? static_cast<size_t>(D + 1) * kRopePairs * (sizeof(double2) + sizeof(float2)) : 0;
}
__device__ __forceinline__ const float2* rope_table_f32(const double2* tab, int D) {
  return reinterpret_cast<const float2*>(tab + (D + 1) * kRopePairs);
}
inline void set_rope(BatchArgs& a, float rope_theta) {
  a.theta = static_cast<double>(rope_theta);
  for (int c = 0; c < kRopePairs; ++c) a.freq[c] = a.theta > 0.0 ? std::pow(a.theta, -2.0 * c / HD) : 0.0;
}
// f: this thread's pair frequency, freq[threadIdx.x % 64], loaded by the
// caller ahead of its bulk loads (a load issued behind them would wait for
// them).
__device__ __forceinline__ void rope_table(double2* tab, int D, int L, double f) {
  const int c = threadIdx.x % kRopePairs;
  for (int d = threadIdx.x / kRopePairs; d <= D; d += blockDim.x / kRopePairs) {
    const double pos = static_cast<double>(L) + static_cast<double>(d);
    double sn, cs;
    sincos(pos * f, &sn, &cs);
    tab[d * kRopePairs + c] = make_double2(cs, sn);
    reinterpret_cast<float2*>(tab + (D + 1) * kRopePairs)[d * kRopePairs + c] =
        make_float2(static_cast<float>(cs), static_cast<float>(sn));
  }
}

// Turns the 8 pairs (c0 + e, c0 + e + 64), e < 8, whose halves lo / hi hold
// (bf16), by the angles at t[c0 .. c0 + 7] (t = the position's table row):
// lo cos - hi sin and hi cos + lo sin in fp64 (each product rounded, then
// the sum: no fused multiply-add), each rounded to bf16 once.
__device__ __forceinline__ void rope_pairs(u32x4& lo, u32x4& hi, const double2* t) {
#pragma clang fp contract(off)
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t nl = 0u, nh = 0u;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const double2 a = t[2 * w + h];
      const double x = bf16_to_f64(static_cast<uint16_t>(lo[w] >> (16 * h)));
      const double y = bf16_to_f64(static_cast<uint16_t>(hi[w] >> (16 * h)));
      nl |= f64_to_bf16_rne(x * a.x - y * a.y) << (16 * h);
      nh |= f64_to_bf16_rne(y * a.x + x * a.y) << (16 * h);
    }
    lo[w] = nl;
    hi[w] = nh;
  }
}

// The same turn in fp32 with fp32 angles, rounded to bf16 by the hardware
// (for the queries, which only enter bf16 products: the cache keeps the
// fp64 form's keys).
__device__ __forceinline__ void rope_pairs_f32(u32x4& lo, u32x4& hi, const float2* t) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float2 a0 = t[2 * w], a1 = t[2 * w + 1];
    const float x0 = bf16_lo(lo[w]), x1 = bf16_hi(lo[w]);
    const float y0 = bf16_lo(hi[w]), y1 = bf16_hi(hi[w]);
    lo[w] = __builtin_bit_cast(uint32_t, __builtin_convertvector(
                                             (f32x2{x0 * a0.x - y0 * a0.y, x1 * a1.x - y1 * a1.y}), bf16x2));
    hi[w] = __builtin_bit_cast(uint32_t, __builtin_convertvector(
                                             (f32x2{y0 * a0.x + x0 * a0.y, y1 * a1.x + x1 * a1.y}), bf16x2));
  }
}

// One half of a pair whose other half sits in lane ^ 8 (a key row loaded as
// 16 lanes x 16 bytes: chunk m holds dims 8m .. 8m + 7): the rotated chunk,
// only this lane's half computed -- mine cos - other sin for the first half,
// mine cos + other sin for the second (the same rounded steps as
// rope_pairs).  Every lane must call it (shuffles); `on` selects the lanes
// that rotate.
__device__ __forceinline__ u32x4 rope_half(const u32x4& mine, int m, bool on, const double2* t) {
#pragma clang fp contract(off)
  u32x4 other;
#pragma unroll
  for (int w = 0; w < 4; ++w) other[w] = static_cast<uint32_t>(__shfl_xor(static_cast<int>(mine[w]), 8, 64));
  if (!on) return mine;
  const double2* a = t + 8 * (m & 7);
  u32x4 out;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t r = 0u;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const double2 cs = a[2 * w + h];
      const double x = bf16_to_f64(static_cast<uint16_t>(mine[w] >> (16 * h)));
      const double y = bf16_to_f64(static_cast<uint16_t>(other[w] >> (16 * h)));
      const double sn = m < 8 ? -cs.y : cs.y;
      r |= f64_to_bf16_rne(x * cs.x + y * sn) << (16 * h);
    }
    out[w] = r;
  }
  return out;
}

// ---------------------------------------------------------------- attend --

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One query tile per workgroup (trees of up to 32 query rows per KV head);
// the per-tile state below is written for NT tiles held by every wave.
// DEVB: a device-planned batch (its own instantiation, so the host-planned
// and single device-planned forms keep their registers).
template <bool DEVB>
__global__ __launch_bounds__(kAttnThreads) void tree_attn_kernel(BatchArgs p) {
  constexpr int NT = 1;
  // blockIdx -> sequence, then (kv head, split) group and query-tile group;
  // the query groups of one (head, split) land on the same XCD (dispatch is
  // round-robin over 8 XCDs and every sequence's range starts at a multiple
  // of 8), so their K/V reads share that XCD's L2.
  const int b = seq_of(p, static_cast<int>(blockIdx.x), [](const SeqPlan& q) { return q.item0; });
  const SeqPlan sq = DEVB ? resolve_batch(p, b) : resolve(p, b);
  if (sq.T == 0) return;
  if (DEVB ? sq.nt != NT : (p.dev && tree_tiles(p.G, sq.T) != NT)) return;   // another instance's
  const int bid = blockIdx.x - sq.item0;
  const int qg = (bid >> 3) % sq.nqg;
  const int gc = ((bid >> 3) / sq.nqg) * 8 + (bid & 7);
  if (gc >= p.Hkv * sq.nsplit) return;
  const int g = gc / sq.nsplit, split = gc % sq.nsplit;
  const int T = sq.T, L = sq.L, nkeys = sq.L + sq.T, rows_pad = sq.rows_pad;
  const int nsplit = sq.nsplit;
  const int qt0 = qg * NT;   // first query tile of the group

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 31, lh = lane >> 5;
  const int GT = p.G * T;
  constexpr int QR = NT * kQTile;   // query rows of a group

  // LDS: the tiles' Q fragments and per-wave V^T tiles during the loop, one
  // region reused for the wave merge after it
  constexpr int kQfBytes = NT * 8 * 64 * 16;
  constexpr int kVtBytes = HD * VT_LD * 2;                           // 9216
  constexpr int OLD = HD + 4;                                         // merge row stride (floats)
  constexpr int kMergeBytes = 2 * kQTile * OLD * 4;                  // 33792: two wave slots
  constexpr int kLoopBytes = kQfBytes + kAttnWaves * kVtBytes;
  constexpr int kLdsBytes = kMergeBytes > kLoopBytes ? kMergeBytes : kLoopBytes;
  __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsBytes];
  __shared__ uint32_t s_mask[QR][ENTMTP_MASK_WORDS + 1];
  __shared__ float s_m[kAttnWaves][QR], s_l[kAttnWaves][QR];
  __shared__ float s_sc[kAttnWaves][QR];   // each wave's factor to the common max
  __shared__ float s_M[QR], s_L[QR];        // a row's common max and sum
  extern __shared__ __attribute__((aligned(16))) double2 s_rope[];   // angles of the tree's positions
  u32x4 (*s_qf)[8][64] = reinterpret_cast<u32x4 (*)[8][64]>(lds);   // [NT][s][lane]
  uint32_t* vt = reinterpret_cast<uint32_t*>(lds + kQfBytes + wave * kVtBytes);  // [HD][VT_LD/2]

  const size_t head_off = static_cast<size_t>(g) * p.cap * HD;
  const uint16_t* kbase = sq.kc + head_off;
  const uint16_t* vbase = sq.vc + head_off;
  const float c = p.scale_log2;
  const int nblocks = (nkeys + KB - 1) / KB;
  const int blk_lo = split * sq.bps;
  const int blk_hi = min(nblocks, blk_lo + sq.bps);

  // K/V of one block into registers: prefix keys from the cache, the tree's
  // keys (slots L and up, not yet rotated) and values from the step's
  // inputs.  Keys past the end are clamped to the last key (finite data
  // whose probabilities are zero), so every load is unconditional and the
  // compiler's wait counts stay exact.
  auto krow = [&](int key) {
    return key < L ? kbase + static_cast<size_t>(key) * HD
                   : p.kt + (static_cast<size_t>(sq.row0 + key - L) * p.Hkv + g) * HD;
  };
  auto vrow = [&](int key) {
    return key < L ? vbase + static_cast<size_t>(key) * HD
                   : p.vt + (static_cast<size_t>(sq.row0 + key - L) * p.Hkv + g) * HD;
  };
  auto load_k = [&](int blk, u32x4 (&kf)[8]) {
    const int kb = blk * KB;
    const int key = min(kb + li, nkeys - 1);
    const uint16_t* kp = krow(key) + 8 * lh;
#pragma unroll
    for (int s = 0; s < 8; ++s) kf[s] = *reinterpret_cast<const u32x4*>(kp + 16 * s);
  };
  auto load_v = [&](int blk, u32x4 (&va)[4], u32x4 (&vb)[4]) {
    const int kb = blk * KB;
    const int last = nkeys - 1;
    // V: key pairs (2pp, 2pp+1) x 8-dim chunk m
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int u = lane + 64 * k;
      const int pp = u & 15, m = u >> 4;
      const int k0 = min(kb + 2 * pp, last), k1 = min(kb + 2 * pp + 1, last);
      va[k] = *reinterpret_cast<const u32x4*>(vrow(k0) + 8 * m);
      vb[k] = *reinterpret_cast<const u32x4*>(vrow(k1) + 8 * m);
    }
  };
  // the first query group's workgroups keep the tree's keys and values in
  // the cache (slots L .. L + T - 1) for the steps after this one
  const bool keeper = qg == 0;
  uint16_t* const kc_head = sq.kc + head_off;
  uint16_t* const vc_head = sq.vc + head_off;

  // Q^T B-operand fragments, the same for the four waves (they split keys,
  // not queries), staged once in LDS: lane (query li, half lh) of tile t
  // reads d = 16s + 8lh + e from slot [t][s][lane].  Query row r of KV head
  // g is (head g * G + r / T, node r % T); thread (s, ln) loads chunks s and
  // s + 4 of its row (the two halves of pairs 16s + 8lh + e).  These small
  // loads (and the masks, the depth and the pair frequency) are requested
  // first and unconditionally (rows past the tree read row 0 and are never
  // stored): behind the waves' first K/V blocks they would wait for every
  // workgroup's burst.
  static_assert(NT * 4 * 64 == kAttnThreads, "one thread per pair of Q chunks");
  const int qs = (tid >> 6) & 3, qhl = (tid >> 5) & 1;
  const int qrow = qt0 * kQTile + li;
  const bool qlive = qrow < GT;
  const int qnode = qlive ? qrow % T : 0;
  u32x4 qlo, qhi;
  {
    const uint16_t* qp = p.q + (static_cast<size_t>(sq.row0 + qnode) * p.Hq + g * p.G + (qlive ? qrow / T : 0)) * HD +
                         8 * qhl + 16 * qs;
    qlo = *reinterpret_cast<const u32x4*>(qp);
    qhi = *reinterpret_cast<const u32x4*>(qp + HD / 2);
  }
  const int qdepth = sq.depth[qnode];
  static_assert(QR * ENTMTP_MASK_WORDS == kAttnThreads, "one mask word per thread");
  const int mrow = qt0 * kQTile + tid / ENTMTP_MASK_WORDS;
  const uint32_t mword = sq.mask[(mrow < GT ? mrow % T : 0) * ENTMTP_MASK_WORDS + tid % ENTMTP_MASK_WORDS];
  const double freq = p.freq[tid % kRopePairs];

  // the wave's first block is requested before the rest of the prologue, so
  // its latency overlaps the staging of the queries
  const bool active = blk_lo + wave < blk_hi;
  u32x4 kA[8], kB[8], v0[4], v1[4];
  int cur = blk_lo + wave;
  if (active) {
    load_k(cur, kA);
    load_v(cur, v0, v1);
  }

  // ancestor masks of the group's query rows (padding rows see every key),
  // the angle table, and the rotated Q fragments into LDS
  s_mask[tid / ENTMTP_MASK_WORDS][tid % ENTMTP_MASK_WORDS] = mrow < GT ? mword : 0xFFFFFFFFu;
  const bool rope = p.theta > 0.0;
  if (rope) {
    rope_table(s_rope, sq.D, L, freq);
    __syncthreads();
    if (qlive) rope_pairs_f32(qlo, qhi, rope_table_f32(s_rope, sq.D) + qdepth * kRopePairs + 16 * qs + 8 * qhl);
  }
  s_qf[0][qs][lane] = qlive ? qlo : u32x4{0u, 0u, 0u, 0u};
  s_qf[0][qs + 4][lane] = qlive ? qhi : u32x4{0u, 0u, 0u, 0u};
  __syncthreads();

  // running (max, sum) per query in base-2 scaled units and the output
  // accumulators, per tile.  The max is raised lazily: the reference m stays
  // until a block's maximum exceeds it by more than kLazyLog2, so that the
  // accumulators are rescaled only a few times per row instead of per block
  // (probabilities relative to m then reach at most 2^kLazyLog2).
  float m_run[NT], l_run[NT];
  f32x16 o[NT][4];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][ct][r] = 0.f;
  }

  // a block's V into this wave's V^T tile: word (dim, key pair) packs the
  // pair's two bf16 values of that dim (and the tree's values into the cache)
  auto stage_v = [&](int blk, const u32x4 (&va)[4], const u32x4 (&vb)[4]) {
    if (keeper && blk * KB + KB > L) {
      const int kb = blk * KB;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int u = lane + 64 * k;
        const int pp = u & 15, m = u >> 4;
        const int k0 = kb + 2 * pp, k1 = k0 + 1;
        if (k0 >= L && k0 < nkeys) *reinterpret_cast<u32x4*>(vc_head + static_cast<size_t>(k0) * HD + 8 * m) = va[k];
        if (k1 >= L && k1 < nkeys) *reinterpret_cast<u32x4*>(vc_head + static_cast<size_t>(k1) * HD + 8 * m) = vb[k];
      }
    }
    wave_lds_sync();  // previous block's V^T reads are done
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int u = lane + 64 * k;
      const int pp = u & 15, m = u >> 4;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t a = va[k][w], bw = vb[k][w];
        // dims 8m + 2w (low halves) and 8m + 2w + 1 (high halves)
        vt[(8 * m + 2 * w) * (VT_LD / 2) + pp] = __builtin_amdgcn_perm(bw, a, 0x05040100u);
        vt[(8 * m + 2 * w + 1) * (VT_LD / 2) + pp] = __builtin_amdgcn_perm(bw, a, 0x07060302u);
      }
    }
  };

  // scores of one tile -> its probabilities as the B operand of the PV
  // product (bf16), with the lazy rescale of the tile's accumulators.
  // Lane (query li, half lh) holds keys n = 8*(r/4) + 4*lh + r%4 of the block.
  auto softmax = [&](int t, f32x16& sacc, int kb, bool plain, bf16x8 (&pf)[2]) {
    float bmax = -INFINITY;
    if (plain) {   // the whole block lies in the prefix: every key is visible
#pragma unroll
      for (int r = 0; r < 16; ++r) bmax = fmaxf(bmax, sacc[r]);
    } else {
      // 32-key window of the query's visibility: prefix keys, then the
      // ancestor bitmask from position L on
      uint32_t win = 0xFFFFFFFFu;
      const int rel = kb - L;
      const uint32_t* mrow = s_mask[t * kQTile + li];
      if (rel < 0) {
        const int npre = -rel;
        win = (0xFFFFFFFFu >> (32 - npre)) | (mrow[0] << npre);
      } else {
        const int wi = rel >> 5, sh = rel & 31;
        const uint32_t lo = mrow[wi];
        const uint32_t hi = wi + 1 < ENTMTP_MASK_WORDS ? mrow[wi + 1] : 0u;
        win = sh ? (lo >> sh) | (hi << (32 - sh)) : lo;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = 8 * (r >> 2) + 4 * lh + (r & 3);
        const bool vis = ((win >> n) & 1u) && (kb + n < nkeys);
        sacc[r] = vis ? sacc[r] : -INFINITY;
        bmax = fmaxf(bmax, sacc[r]);
      }
    }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float mb = bmax * c;   // -inf stays -inf (c > 0)
    const bool need = mb > m_run[t] + kLazyLog2;
    if (__any(need)) {   // uniform branch: rare once the row maximum has settled
      const float mn = need ? mb : m_run[t];
      const float alpha = !need ? 1.f : (m_run[t] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[t] - mn));
      l_run[t] *= alpha;
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[t][ct][r] *= alpha;
      m_run[t] = mn;
    }
    // with m still -inf every key so far is hidden from the query: p = 0
    const float mneg = m_run[t] == -INFINITY ? 0.f : -m_run[t];
    float pr[16];
    float rsum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      pr[r] = __builtin_amdgcn_exp2f(fmaf(sacc[r], c, mneg));
      rsum += pr[r];
    }
    rsum += __shfl_xor(rsum, 32, 64);
    l_run[t] += rsum;
    // P^T as B operand: step u covers keys 16u..16u+15; element e of lane
    // (query li, half lh) is key 16u + 4lh + e (e < 4) or 16u + 8 + 4lh + e-4
    // -- exactly accumulator entries 8u .. 8u+7.
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(
                                               (f32x2{pr[8 * u + 2 * e], pr[8 * u + 2 * e + 1]}), bf16x2));
      pf[u] = as_bf16x8(w);
    }
  };

  // the block's scores, softmax and P V for the group's tiles (V from the
  // staged tile, each V^T fragment read once for all tiles)
  auto attend = [&](int blk, u32x4 (&kf)[8]) {
    const int kb = blk * KB;
    const bool plain = kb + KB <= L;
    if (!plain) {   // the tree's keys: rotate, and keep them in the cache
      const int key = min(kb + li, nkeys - 1);
      if (key >= L) {
        if (rope) {
          const double2* tr = s_rope + sq.depth[key - L] * kRopePairs + 8 * lh;
#pragma unroll
          for (int s = 0; s < 4; ++s) rope_pairs(kf[s], kf[s + 4], tr + 16 * s);
        }
        if (keeper && kb + li < nkeys) {
#pragma unroll
          for (int s = 0; s < 8; ++s)
            *reinterpret_cast<u32x4*>(kc_head + static_cast<size_t>(key) * HD + 8 * lh + 16 * s) = kf[s];
        }
      }
    }
    f32x16 sacc[NT];
    bf16x8 pf[NT][2];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      // S^T[key][query] = K Q^T
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s)
        sacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[s]), as_bf16x8(s_qf[t][s][lane]),
                                                        sacc[t], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      softmax(t, sacc[t], kb, plain, pf[t]);
    }
    wave_lds_sync();  // V^T tile written by every lane
    // O^T[dim][query] += V^T P^T; A operand lane (dim li of tile ct, half lh)
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const uint32_t* row = vt + (32 * ct + li) * (VT_LD / 2);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint2 x0 = *reinterpret_cast<const uint2*>(row + 8 * u + 2 * lh);
        const uint2 x1 = *reinterpret_cast<const uint2*>(row + 8 * u + 4 + 2 * lh);
        const u32x4 w = {x0.x, x0.y, x1.x, x1.y};
#pragma unroll
        for (int t = 0; t < NT; ++t)
          o[t][ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(w), pf[t][u], o[t][ct], 0, 0, 0);
      }
    }
  };

  // K two deep (block b+4 streams in while block b is multiplied); V one
  // deep, the next block's loads issued as soon as this block's V is in its
  // LDS tile.  (The loads after a wave's last block re-read that block, an
  // L2 hit.)
  if (active) {
    while (true) {
      const int nb = cur + kAttnWaves;
      const int nbc = nb < blk_hi ? nb : cur;
      load_k(nbc, kB);
      stage_v(cur, v0, v1);
      load_v(nbc, v0, v1);
      attend(cur, kA);
      if (nb >= blk_hi) break;
      const int nb2 = nb + kAttnWaves;
      const int nb2c = nb2 < blk_hi ? nb2 : nb;
      load_k(nb2c, kA);
      stage_v(nb, v0, v1);
      load_v(nb2c, v0, v1);
      attend(nb, kB);
      if (nb2 >= blk_hi) break;
      cur = nb2;
    }
  }

  // ---- merge the four waves, tile by tile: each wave rescales to the
  // common reference max; waves 2 and 3 hand their sums to 0 and 1 through
  // two LDS slots, 0 and 1 write the pair sums back, and all threads combine
  // the two slots into the output (float4 rows, no more LDS than the loop's)
  __syncthreads();  // every wave is done with its Q fragments and V^T tile
  if (lh == 0) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      s_m[wave][t * kQTile + li] = m_run[t];
      s_l[wave][t * kQTile + li] = l_run[t];
    }
  }
  __syncthreads();
  // per row, once: the common max, each wave's factor to it, and the sum
  if (tid < QR) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, s_m[w][tid]);
    float lsum = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      const float sc = (s_m[w][tid] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(s_m[w][tid] - M);
      s_sc[w][tid] = sc;
      lsum += s_l[w][tid] * sc;
    }
    s_M[tid] = M;
    s_L[tid] = lsum;
  }
  __syncthreads();
  float* ored = reinterpret_cast<float*>(lds);  // [slot][query][OLD]
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const float myscale = s_sc[wave][t * kQTile + li];
    // lane (query li, half lh) holds dims 32ct + 8j + 4lh + i in o[t][ct][4j + i]
    auto slot_at = [&](int slot, int ct, int j) {
      return reinterpret_cast<float4*>(ored + (slot * kQTile + li) * OLD + 32 * ct + 8 * j + 4 * lh);
    };
    if (t > 0) __syncthreads();   // the previous tile's slots are read out
    if (wave >= 2) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *slot_at(wave - 2, ct, j) = make_float4(o[t][ct][4 * j] * myscale, o[t][ct][4 * j + 1] * myscale,
                                                  o[t][ct][4 * j + 2] * myscale, o[t][ct][4 * j + 3] * myscale);
    }
    __syncthreads();
    if (wave < 2) {
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float4* sl = slot_at(wave, ct, j);
          const float4 x = *sl;
          *sl = make_float4(x.x + o[t][ct][4 * j] * myscale, x.y + o[t][ct][4 * j + 1] * myscale,
                            x.z + o[t][ct][4 * j + 2] * myscale, x.w + o[t][ct][4 * j + 3] * myscale);
        }
    }
    __syncthreads();
    // thread -> (query q, four dims): 32 x 32 float4 items, four per thread
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int x = tid + kAttnThreads * i;
      const int q = x >> 5, d4 = 4 * (x & 31);
      const int row = (qt0 + t) * kQTile + q;
      if (row >= GT) continue;
      const int sr = t * kQTile + q;
      const float Mq = s_M[sr], lsum = s_L[sr];
      const float4 s0 = *reinterpret_cast<const float4*>(ored + q * OLD + d4);
      const float4 s1 = *reinterpret_cast<const float4*>(ored + (kQTile + q) * OLD + d4);
      const float4 os = make_float4(s0.x + s1.x, s0.y + s1.y, s0.z + s1.z, s0.w + s1.w);
      if (nsplit == 1) {
        const int gh = row / T, node = row % T;
        const int h = g * p.G + gh;
        uint2 pk;
        pk.x = f32_to_bf16_rne(os.x / lsum) | (f32_to_bf16_rne(os.y / lsum) << 16);
        pk.y = f32_to_bf16_rne(os.z / lsum) | (f32_to_bf16_rne(os.w / lsum) << 16);
        *reinterpret_cast<uint2*>(p.out + (static_cast<size_t>(sq.row0 + node) * p.Hq + h) * HD + d4) = pk;
      } else {
        const size_t prow = sq.part_off + (static_cast<size_t>(split) * p.Hkv + g) * rows_pad + row;
        const float il = lsum > 0.f ? 1.f / lsum : 0.f;   // 0: no key of the split is visible
        uint2 pk;
        pk.x = f32_to_bf16_rne(os.x * il) | (f32_to_bf16_rne(os.y * il) << 16);
        pk.y = f32_to_bf16_rne(os.z * il) | (f32_to_bf16_rne(os.w * il) << 16);
        *reinterpret_cast<uint2*>(p.part_o + prow * HD + d4) = pk;
        if (d4 == 0) {
          p.part_ml[prow * 2 + 0] = Mq;
          p.part_ml[prow * 2 + 1] = lsum;
        }
      }
    }
  }
}

// Four query tiles per workgroup, one per wave (trees with more than 32
// query rows per KV head; waves past the tree's last tile only load): the four waves walk the same key blocks, which
// the workgroup stages once in LDS -- K as rows, V transposed -- from
// coalesced loads (16 lanes per 256-byte key row), double-buffered with one
// barrier per block and two blocks in flight in registers, so a KV block is
// read once per 128 query rows.  Each wave keeps its own tile's Q fragments,
// softmax state and output, so no cross-wave merge is needed.
constexpr int KROW = HD + 8;   // bf16 per staged K row (16-byte pad: rows 4 banks apart)

template <bool DEVB>
__global__ __launch_bounds__(kAttnThreads, 2) void tree_attn_q4_kernel(BatchArgs p) {
  const int b = seq_of(p, static_cast<int>(blockIdx.x), [](const SeqPlan& q) { return q.item0; });
  const SeqPlan sq = DEVB ? resolve_batch(p, b) : resolve(p, b);
  if (sq.T == 0) return;
  if (DEVB ? sq.nt != 4 : (p.dev && tree_tiles(p.G, sq.T) != 4)) return;   // another instance's
  const int bid = blockIdx.x - sq.item0;
  const int qg = (bid >> 3) % sq.nqg;
  const int gc = ((bid >> 3) / sq.nqg) * 8 + (bid & 7);
  if (gc >= p.Hkv * sq.nsplit) return;
  const int g = gc / sq.nsplit, split = gc % sq.nsplit;
  const int T = sq.T, L = sq.L, nkeys = sq.L + sq.T, rows_pad = sq.rows_pad;
  const int nsplit = sq.nsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 31, lh = lane >> 5;
  const int GT = p.G * T;
  const int qt = qg * 4 + wave;           // this wave's query tile
  const bool live = qt < sq.nqt;          // (uniform per wave)
  constexpr int QR = 4 * kQTile;

  __shared__ __attribute__((aligned(16))) uint16_t s_k[2][KB][KROW];
  __shared__ __attribute__((aligned(16))) uint32_t s_vt[2][HD * (VT_LD / 2)];
  __shared__ uint32_t s_mask[QR][ENTMTP_MASK_WORDS + 1];
  extern __shared__ __attribute__((aligned(16))) double2 s_rope[];   // angles of the tree's positions

  const size_t head_off = static_cast<size_t>(g) * p.cap * HD;
  uint16_t* const kc_head = sq.kc + head_off;
  uint16_t* const vc_head = sq.vc + head_off;
  const uint16_t* kbase = kc_head;
  const uint16_t* vbase = vc_head;
  const float c = p.scale_log2;
  const int nblocks = (nkeys + KB - 1) / KB;
  const int blk_lo = split * sq.bps;
  const int blk_hi = min(nblocks, blk_lo + sq.bps);
  const int nb = blk_hi - blk_lo;
  const bool rope = p.theta > 0.0;
  // the first query group's workgroups keep the tree's keys (rotated) and
  // values in the cache (slots L .. L + T - 1) for the steps after this one
  const bool keeper = qg == 0;

  // prefix keys from the cache, the tree's keys and values from the inputs
  auto krow = [&](int key) {
    return key < L ? kbase + static_cast<size_t>(key) * HD
                   : p.kt + (static_cast<size_t>(sq.row0 + key - L) * p.Hkv + g) * HD;
  };
  auto vrow = [&](int key) {
    return key < L ? vbase + static_cast<size_t>(key) * HD
                   : p.vt + (static_cast<size_t>(sq.row0 + key - L) * p.Hkv + g) * HD;
  };
  // cooperative loads of one block: K unit u = tid + 256 j -> key u / 16,
  // 16-byte chunk u % 16; V unit tid -> key pair tid / 16, 8-dim chunk
  // tid % 16 (both keys of the pair).  Keys past the end clamp to the last.
  auto gload = [&](int i, u32x4 (&kr)[2], u32x4& va, u32x4& vb) {
    const int kb = (blk_lo + min(i, nb - 1)) * KB;
    const int last = nkeys - 1;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int u = tid + kAttnThreads * j;
      const int key = min(kb + (u >> 4), last);
      kr[j] = *reinterpret_cast<const u32x4*>(krow(key) + 8 * (u & 15));
    }
    const int m = tid & 15, pp = tid >> 4;
    const int k0 = min(kb + 2 * pp, last), k1 = min(kb + 2 * pp + 1, last);
    va = *reinterpret_cast<const u32x4*>(vrow(k0) + 8 * m);
    vb = *reinterpret_cast<const u32x4*>(vrow(k1) + 8 * m);
  };
  // block i's registers into LDS buffer buf; a block that holds tree keys
  // rotates them first (the pair's other half sits in lane ^ 8) and the
  // keeper writes them and their values to the cache
  auto stage = [&](int buf, int i, u32x4 (&kr)[2], const u32x4& va, const u32x4& vb) {
    const int kb = (blk_lo + min(i, nb - 1)) * KB;
    if (kb + KB > L) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int u = tid + kAttnThreads * j;
        const int key = kb + (u >> 4);
        const int kk = min(key, nkeys - 1);
        if (rope)
          kr[j] = rope_half(kr[j], u & 15, kk >= L, s_rope + sq.depth[max(kk - L, 0)] * kRopePairs);
        if (keeper && key >= L && key < nkeys)
          *reinterpret_cast<u32x4*>(kc_head + static_cast<size_t>(key) * HD +
                                    8 * (u & 15)) = kr[j];
      }
      const int m = tid & 15, pp = tid >> 4;
      const int k0 = kb + 2 * pp, k1 = k0 + 1;
      if (keeper && k0 >= L && k0 < nkeys)
        *reinterpret_cast<u32x4*>(vc_head + static_cast<size_t>(k0) * HD + 8 * m) = va;
      if (keeper && k1 >= L && k1 < nkeys)
        *reinterpret_cast<u32x4*>(vc_head + static_cast<size_t>(k1) * HD + 8 * m) = vb;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int u = tid + kAttnThreads * j;
      *reinterpret_cast<u32x4*>(&s_k[buf][u >> 4][8 * (u & 15)]) = kr[j];
    }
    const int m = tid & 15, pp = tid >> 4;
    uint32_t* vt = s_vt[buf];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      vt[(8 * m + 2 * w) * (VT_LD / 2) + pp] = __builtin_amdgcn_perm(vb[w], va[w], 0x05040100u);
      vt[(8 * m + 2 * w + 1) * (VT_LD / 2) + pp] = __builtin_amdgcn_perm(vb[w], va[w], 0x07060302u);
    }
  };

  // The small loads go first (this wave's Q fragments, its rows' depths and
  // the group's masks, all unconditional: rows past the tree read row 0 and
  // are never stored): requested after the first two K/V blocks they waited
  // behind every workgroup's 32 KB burst (measured: a 6 us prologue).
  // Query row r of KV head g is (head g * G + r / T, node r % T); chunks s
  // and s + 4 hold the two halves of pairs 16s + 8lh + e.
  u32x4 qf[8];
  const int qrow = qt * kQTile + li;
  const bool qlive = qrow < GT;
  const int qnode = qlive ? qrow % T : 0;
  {
    const uint16_t* qp = p.q + (static_cast<size_t>(sq.row0 + qnode) * p.Hq + g * p.G + (qlive ? qrow / T : 0)) * HD +
                         8 * lh;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = *reinterpret_cast<const u32x4*>(qp + 16 * s);
  }
  const int qdepth = sq.depth[qnode];
  constexpr int kMaskPer = QR * ENTMTP_MASK_WORDS / kAttnThreads;
  static_assert(kMaskPer * kAttnThreads == QR * ENTMTP_MASK_WORDS, "mask words fill the threads");
  uint32_t mw[kMaskPer];
#pragma unroll
  for (int j = 0; j < kMaskPer; ++j) {
    const int u = tid + kAttnThreads * j;
    const int mrow = qg * QR + u / ENTMTP_MASK_WORDS;
    mw[j] = sq.mask[(mrow < GT ? mrow % T : 0) * ENTMTP_MASK_WORDS + u % ENTMTP_MASK_WORDS];
  }
  const double freq = p.freq[tid % kRopePairs];

  u32x4 kA[2], kB[2], vaA, vbA, vaB, vbB;
  gload(0, kA, vaA, vbA);
  gload(1, kB, vaB, vbB);

  // ancestor masks of the group's rows (padding rows see every key), the
  // angle table and this wave's rotated Q fragments, while the blocks arrive
#pragma unroll
  for (int j = 0; j < kMaskPer; ++j) {
    const int u = tid + kAttnThreads * j;
    const int r = u / ENTMTP_MASK_WORDS;
    s_mask[r][u % ENTMTP_MASK_WORDS] = qg * QR + r < GT ? mw[j] : 0xFFFFFFFFu;
  }
  if (rope) {
    rope_table(s_rope, sq.D, L, freq);
    __syncthreads();
    if (qlive) {
      const float2* tr = rope_table_f32(s_rope, sq.D) + qdepth * kRopePairs + 8 * lh;
#pragma unroll
      for (int s = 0; s < 4; ++s) rope_pairs_f32(qf[s], qf[s + 4], tr + 16 * s);
    }
  }
  stage(0, 0, kA, vaA, vbA);
  gload(2, kA, vaA, vbA);
  __syncthreads();

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ct][r] = 0.f;

  // block i of the split from LDS buffer buf: this wave's scores, softmax
  // (lazily raised max, as in tree_attn_kernel) and P V
  auto compute = [&](int i, int buf) {
    if (!live) return;
    const int kb = (blk_lo + i) * KB;
    const bool plain = kb + KB <= L;
    f32x16 sacc;
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const u32x4 kf = *reinterpret_cast<const u32x4*>(&s_k[buf][li][16 * s + 8 * lh]);
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf), as_bf16x8(qf[s]), sacc, 0, 0, 0);
    }
    float bmax = -INFINITY;
    if (plain) {
#pragma unroll
      for (int r = 0; r < 16; ++r) bmax = fmaxf(bmax, sacc[r]);
    } else {
      uint32_t win = 0xFFFFFFFFu;
      const int rel = kb - L;
      const uint32_t* mrow = s_mask[wave * kQTile + li];
      if (rel < 0) {
        const int npre = -rel;
        win = (0xFFFFFFFFu >> (32 - npre)) | (mrow[0] << npre);
      } else {
        const int wi = rel >> 5, sh = rel & 31;
        const uint32_t lo = mrow[wi];
        const uint32_t hi = wi + 1 < ENTMTP_MASK_WORDS ? mrow[wi + 1] : 0u;
        win = sh ? (lo >> sh) | (hi << (32 - sh)) : lo;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = 8 * (r >> 2) + 4 * lh + (r & 3);
        const bool vis = ((win >> n) & 1u) && (kb + n < nkeys);
        sacc[r] = vis ? sacc[r] : -INFINITY;
        bmax = fmaxf(bmax, sacc[r]);
      }
    }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float mb = bmax * c;
    const bool need = mb > m_run + kLazyLog2;
    if (__any(need)) {
      const float mn = need ? mb : m_run;
      const float alpha = !need ? 1.f : (m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - mn));
      l_run *= alpha;
#pragma unroll
      for (int ct = 0; ct < 4; ++ct)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[ct][r] *= alpha;
      m_run = mn;
    }
    const float mneg = m_run == -INFINITY ? 0.f : -m_run;
    float pr[16];
    float rsum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      pr[r] = __builtin_amdgcn_exp2f(fmaf(sacc[r], c, mneg));
      rsum += pr[r];
    }
    rsum += __shfl_xor(rsum, 32, 64);
    l_run += rsum;
    bf16x8 pf[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = __builtin_bit_cast(uint32_t, __builtin_convertvector(
                                               (f32x2{pr[8 * u + 2 * e], pr[8 * u + 2 * e + 1]}), bf16x2));
      pf[u] = as_bf16x8(w);
    }
    const uint32_t* vt = s_vt[buf];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const uint32_t* row = vt + (32 * ct + li) * (VT_LD / 2);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const uint2 x0 = *reinterpret_cast<const uint2*>(row + 8 * u + 2 * lh);
        const uint2 x1 = *reinterpret_cast<const uint2*>(row + 8 * u + 4 + 2 * lh);
        const u32x4 w = {x0.x, x0.y, x1.x, x1.y};
        o[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(w), pf[u], o[ct], 0, 0, 0);
      }
    }
  };

  // block i computes from buffer i & 1 while block i + 1 is staged into the
  // other buffer and block i + 3 streams into the freed registers
  for (int i = 0;; i += 2) {
    compute(i, 0);
    if (i + 1 >= nb) break;
    stage(1, i + 1, kB, vaB, vbB);
    gload(i + 3, kB, vaB, vbB);
    __syncthreads();
    compute(i + 1, 1);
    if (i + 2 >= nb) break;
    stage(0, i + 2, kA, vaA, vbA);
    gload(i + 4, kA, vaA, vbA);
    __syncthreads();
  }

  // this wave's tile: the output (one split) or its partial
  if (!live) return;
  const int row = qt * kQTile + li;
  if (row >= GT) return;
  if (nsplit == 1) {
    const int gh = row / T, node = row % T;
    uint16_t* dst = p.out + (static_cast<size_t>(sq.row0 + node) * p.Hq + g * p.G + gh) * HD;
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint2 pk;
        pk.x = f32_to_bf16_rne(o[ct][4 * j] / l_run) | (f32_to_bf16_rne(o[ct][4 * j + 1] / l_run) << 16);
        pk.y = f32_to_bf16_rne(o[ct][4 * j + 2] / l_run) | (f32_to_bf16_rne(o[ct][4 * j + 3] / l_run) << 16);
        *reinterpret_cast<uint2*>(dst + 32 * ct + 8 * j + 4 * lh) = pk;
      }
  } else {
    const size_t prow = sq.part_off + (static_cast<size_t>(split) * p.Hkv + g) * rows_pad + row;
    uint16_t* dst = p.part_o + prow * HD;
    const float il = l_run > 0.f ? 1.f / l_run : 0.f;   // 0: no key of the split is visible
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint2 pk;
        pk.x = f32_to_bf16_rne(o[ct][4 * j] * il) | (f32_to_bf16_rne(o[ct][4 * j + 1] * il) << 16);
        pk.y = f32_to_bf16_rne(o[ct][4 * j + 2] * il) | (f32_to_bf16_rne(o[ct][4 * j + 3] * il) << 16);
        *reinterpret_cast<uint2*>(dst + 32 * ct + 8 * j + 4 * lh) = pk;
      }
    if (lh == 0) {
      p.part_ml[prow * 2 + 0] = m_run;
      p.part_ml[prow * 2 + 1] = l_run;
    }
  }
}

// ----------------------------------------------------------------- merge --

// One half-wavefront per output row (kMergeRows rows per block): lane c <
// nsplit reads split c's (max, sum) and every lane then requests its four
// dims of the first kMergeBatch splits' partial outputs at once (one memory
// latency instead of one per four splits: the kernel's time was those
// rounds), the group reduces the (max, sum) pairs to the common max and the
// normalised split weights, and combines; splits past the batch follow four
// at a time.
constexpr int kMergeRows = 8;
constexpr int kMergeBatch = 16;   // splits whose partials are requested together
constexpr int kMergeThreads = 32 * kMergeRows;
static_assert(kMaxSplits <= 32, "a half-wavefront holds one lane per split");

template <bool DEVB>
__global__ __launch_bounds__(kMergeThreads) void attn_merge_kernel(BatchArgs p) {
  const int b = seq_of(p, static_cast<int>(blockIdx.x), [](const SeqPlan& q) { return q.merge0; });
  const SeqPlan sq = DEVB ? resolve_batch(p, b) : resolve(p, b);
  if (sq.nsplit == 1 || sq.T == 0) return;   // written by the attend kernel, or nothing to do
  const int GT = p.G * sq.T;
  const int local = (blockIdx.x - sq.merge0) * kMergeRows + (threadIdx.x >> 5);
  if (local >= p.Hkv * GT) return;   // past the last row (device-planned grids cover the largest tree)
  const int g = local / GT, row = local % GT;
  const int lane = threadIdx.x & 31;
  const int nsplit = sq.nsplit;
  auto prow_of = [&](int c) {
    return sq.part_off + (static_cast<size_t>(c) * p.Hkv + g) * sq.rows_pad + row;
  };
  float mc = -INFINITY, lc = 0.f;
  if (lane < nsplit) {
    const float2 ml = *reinterpret_cast<const float2*>(p.part_ml + prow_of(lane) * 2);
    mc = ml.x;
    lc = ml.y;
  }
  const int d4 = 4 * lane;
  uint2 ob[kMergeBatch];
#pragma unroll
  for (int c = 0; c < kMergeBatch; ++c)
    ob[c] = *reinterpret_cast<const uint2*>(p.part_o + prow_of(min(c, nsplit - 1)) * HD + d4);
  float M = mc;
#pragma unroll
  for (int off = 16; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 32));
  const float w = mc == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mc - M);
  float lsum = lc * w;
#pragma unroll
  for (int off = 16; off >= 1; off >>= 1) lsum += __shfl_xor(lsum, off, 32);
  const float wn = w * lc / lsum;   // the split's share of the row
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  auto add = [&](float wc, uint2 v) {
    acc.x += wc * __uint_as_float(v.x << 16);
    acc.y += wc * __uint_as_float(v.x & 0xffff0000u);
    acc.z += wc * __uint_as_float(v.y << 16);
    acc.w += wc * __uint_as_float(v.y & 0xffff0000u);
  };
#pragma unroll
  for (int c = 0; c < kMergeBatch; ++c) add(c < nsplit ? __shfl(wn, c, 32) : 0.f, ob[c]);
  for (int c0 = kMergeBatch; c0 < nsplit; c0 += 4) {   // four splits' loads in flight at a time
    uint2 o[4];
    float wc[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int c = min(c0 + k, nsplit - 1);
      wc[k] = c0 + k < nsplit ? __shfl(wn, c, 32) : 0.f;
      o[k] = *reinterpret_cast<const uint2*>(p.part_o + prow_of(c) * HD + d4);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) add(wc[k], o[k]);
  }
  const int gh = row / sq.T, node = row % sq.T;
  uint2 pk;
  pk.x = f32_to_bf16_rne(acc.x) | (f32_to_bf16_rne(acc.y) << 16);
  pk.y = f32_to_bf16_rne(acc.z) | (f32_to_bf16_rne(acc.w) << 16);
  *reinterpret_cast<uint2*>(p.out + (static_cast<size_t>(sq.row0 + node) * p.Hq + g * p.G + gh) * HD + d4) = pk;
}

// ------------------------------------------------------------------ host --

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

// lds: bytes of the rotation table (rope_lds_bytes of the deepest tree)
template <bool DEVB = false>
void launch_attend(const BatchArgs& a, int items, size_t lds, hipStream_t s) {
  if (a.nt == 4)
    hipLaunchKernelGGL(tree_attn_q4_kernel<DEVB>, dim3(items), dim3(kAttnThreads), lds, s, a);
  else
    hipLaunchKernelGGL(tree_attn_kernel<DEVB>, dim3(items), dim3(kAttnThreads), lds, s, a);
}



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

// Grid sizes of one call.
struct CallShape {
  int rows = 0;          // concatenated tree rows
  int D = 0;             // depth of the deepest tree
  int items = 0;         // attend workgroups
  int merge_blocks = 0;  // merge blocks
  size_t need = 0;       // workspace bytes
};

// Plans the sequences of one call: per-sequence split counts (a lone
// sequence fills the CUs by itself; a batch shares one blocks-per-split
// target sized to about kBatchWgPerCu workgroups per CU), grid ranges and the packed
// workspace layout (output partials, then (max, sum) partials).
CallShape plan_call(const entmtp_bank* bank, int B, const int32_t* topo, const int32_t* L,
                    entmtp_bf16* const* kc, entmtp_bf16* const* vc, int cap, int Hq, int Hkv,
                    BatchArgs& a) {
  a.dev = nullptr;
  a.topos = nullptr;
  a.arena = nullptr;
  a.topo_dev = nullptr;
  a.len_dev = nullptr;
  a.row_off_dev = nullptr;
  a.B = B;
  a.G = Hq / Hkv;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.cap = cap;
  const int cus = device_cus();
  a.cus = cus;
  a.nt = 1;   // the largest tile count any sequence needs
  for (int b = 0; b < B; ++b) {
    const int nt = tree_tiles(a.G, bank->desc[topo[b]].T);
    a.nt = nt > a.nt ? nt : a.nt;
  }
  long long work = 0;   // key-block streams
  for (int b = 0; b < B; ++b) {
    const int T = bank->desc[topo[b]].T;
    const int nqg = query_groups(rows_padded(a.G, T) / kQTile, a.nt);
    work += static_cast<long long>(Hkv) * nqg * ((L[b] + T + KB - 1) / KB);
  }
  const long long per_wg = (work + kBatchWgPerCu * cus - 1) / (kBatchWgPerCu * cus);
  const int target_bps = static_cast<int>(per_wg > kMinBlocksPerSplit ? per_wg : kMinBlocksPerSplit);

  CallShape sh;
  long long part_rows = 0;
  for (int b = 0; b < B; ++b) {
    const TopoDesc& td = bank->desc[topo[b]];
    SeqPlan& q = a.s[b];
    q.kc = kc[b];
    q.vc = vc[b];
    q.mask = bank_ptr<uint32_t>(bank, td.off_mask);
    q.depth = bank_ptr<int>(bank, td.off_depth);
    q.T = td.T;
    q.D = td.D;
    q.L = L[b];
    q.row0 = sh.rows;
    q.rows_pad = rows_padded(a.G, q.T);
    q.nqt = q.rows_pad / kQTile;
    q.nqg = query_groups(q.nqt, a.nt);
    q.nt = a.nt;
    const int nblocks = (q.L + q.T + KB - 1) / KB;
    int ns;
    if (B == 1) {
      ns = split_single(nblocks, Hkv * q.nqg, cus * wg_per_cu(a.nt));
    } else {
      ns = (nblocks + target_bps - 1) / target_bps;
      const int bound = split_bound(nblocks);
      ns = ns < 1 ? 1 : (ns > bound ? bound : ns);
    }
    q.bps = (nblocks + ns - 1) / ns;
    q.nsplit = (nblocks + q.bps - 1) / q.bps;
    q.item0 = sh.items;
    q.merge0 = sh.merge_blocks;
    q.part_off = part_rows;
    sh.rows += q.T;
    sh.D = q.D > sh.D ? q.D : sh.D;
    sh.items += (Hkv * q.nsplit + 7) / 8 * 8 * q.nqg;
    if (q.nsplit > 1) {
      sh.merge_blocks += (Hkv * a.G * q.T + kMergeRows - 1) / kMergeRows;
      part_rows += static_cast<long long>(q.nsplit) * Hkv * q.rows_pad;
    }
  }
  const size_t po = static_cast<size_t>(part_rows) * HD * sizeof(uint16_t);
  const size_t pml = static_cast<size_t>(part_rows) * 2 * 4;
  sh.need = al256(po) + al256(pml);
  return sh;
}

// Points the planned call at its workspace and launches attend and (when
// some sequence has several splits) merge.
int32_t launch_call(BatchArgs& a, const CallShape& sh, void* workspace, hipStream_t s) {
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  long long part_rows = 0;
  for (int b = 0; b < a.B; ++b)
    if (a.s[b].nsplit > 1) part_rows += static_cast<long long>(a.s[b].nsplit) * a.Hkv * a.s[b].rows_pad;
  const size_t po = static_cast<size_t>(part_rows) * HD * sizeof(uint16_t);
  a.part_o = reinterpret_cast<uint16_t*>(ws);
  a.part_ml = reinterpret_cast<float*>(ws + al256(po));
  launch_attend(a, sh.items, rope_lds_bytes(sh.D, a.theta), s);
  if (int32_t rc = launch_status("tree_attn launch")) return rc;
  if (sh.merge_blocks > 0) {
    hipLaunchKernelGGL(attn_merge_kernel<false>, dim3(sh.merge_blocks), dim3(kMergeThreads), 0, s, a);
    if (int32_t rc = launch_status("tree_attn merge launch")) return rc;
  }
  return ENTMTP_OK;
}

size_t workspace_bytes(int T, int Hq, int Hkv, int L) {
  // sized with the largest split count a plan can choose, so the figure
  // never shrinks when T or L grows
  const int G = Hq / Hkv;
  const int rows_pad = rows_padded(G, T);
  const int nblocks = (L + T + KB - 1) / KB;
  const size_t bound = split_bound(nblocks);
  return al256(bound * Hkv * rows_pad * HD * sizeof(uint16_t)) + al256(bound * Hkv * rows_pad * 2 * 4);
}

// Checks shared by the single and batched entry points.
int32_t check_common(int32_t Hq, int32_t Hkv, int32_t d, float scale, float rope_theta,
                     const void* q, const void* k_tree, const void* v_tree, const void* out,
                     const void* workspace) {
  ENTMTP_CHECK_ARG(q && k_tree && v_tree && out && workspace, ENTMTP_EINVAL,
                   "tensor and workspace pointers must be non-NULL");
  ENTMTP_CHECK_ARG(d == HD, ENTMTP_EINVAL, "head dim %d unsupported (built for %d)", d, HD);
  ENTMTP_CHECK_ARG(Hq >= 1 && Hkv >= 1, ENTMTP_EINVAL, "Hq = %d, Hkv = %d must be >= 1", Hq, Hkv);
  ENTMTP_CHECK_ARG(Hq % Hkv == 0, ENTMTP_ERANGE, "Hq = %d is not a multiple of Hkv = %d", Hq, Hkv);
  ENTMTP_CHECK_ARG(Hq / Hkv <= 32, ENTMTP_ERANGE, "query group %d too large", Hq / Hkv);
  ENTMTP_CHECK_ARG(scale > 0.f && scale < INFINITY, ENTMTP_EINVAL, "scale must be positive");
  ENTMTP_CHECK_ARG(rope_theta >= 0.f && rope_theta < INFINITY, ENTMTP_EINVAL,
                   "rope_theta must be >= 0");
  ENTMTP_CHECK_ARG(aligned16(q) && aligned16(k_tree) && aligned16(v_tree) && aligned16(out) &&
                       aligned16(workspace),
                   ENTMTP_EINVAL, "tensors and workspace must be 16-byte aligned");
  return ENTMTP_OK;
}

int32_t check_sequence(const entmtp_bank* bank, int32_t topo, int32_t prefix_len,
                       const void* kc, const void* vc, int32_t cap, int b) {
  if (int32_t rc = check_device_bank(bank, topo)) return rc;
  ENTMTP_CHECK_ARG(kc && vc && aligned16(kc) && aligned16(vc), ENTMTP_EINVAL,
                   "sequence %d: caches must be non-NULL and 16-byte aligned", b);
  ENTMTP_CHECK_ARG(prefix_len >= 0, ENTMTP_EINVAL, "sequence %d: prefix_len = %d < 0", b,
                   prefix_len);
  const int T = bank->desc[topo].T;
  ENTMTP_CHECK_ARG(static_cast<int64_t>(prefix_len) + T <= cap, ENTMTP_ERANGE,
                   "sequence %d: cache capacity %d below prefix_len + T = %d", b, cap,
                   prefix_len + T);
  return ENTMTP_OK;
}

}  // namespace

int32_t attn_device_shape(const entmtp_bank* bank, int Hq, int Hkv, int cap, DevAttnShape* out) {
  const int cus = device_cus();
  const int G = Hq / Hkv;
  DevAttnShape sh;
  for (const TopoDesc& td : bank->desc) {
    sh.T_max = td.T > sh.T_max ? td.T : sh.T_max;
    sh.D_max = td.D > sh.D_max ? td.D : sh.D_max;
    const int nt = tree_tiles(G, td.T);
    const int nqg = query_groups(rows_padded(G, td.T) / kQTile, nt);
    const int max_blocks = (cap + KB - 1) / KB;
    for (int nblocks = 1; nblocks <= max_blocks; ++nblocks) {
      const int ns0 = split_single(nblocks, Hkv * nqg, cus * wg_per_cu(nt));
      const int bps = (nblocks + ns0 - 1) / ns0;
      const int ns = (nblocks + bps - 1) / bps;
      const int items = (Hkv * ns + 7) / 8 * 8 * nqg;
      sh.items[nt] = items > sh.items[nt] ? items : sh.items[nt];
    }
  }
  sh.rows = sh.T_max;
  sh.merge_blocks = (Hkv * G * sh.T_max + kMergeRows - 1) / kMergeRows;
  sh.need = workspace_bytes(sh.T_max, Hq, Hkv, cap);
  *out = sh;
  return ENTMTP_OK;
}

void attn_device_splits(const entmtp_bank* bank, int Hq, int Hkv, DevTopo* topos) {
  const int cus = device_cus();
  const int G = Hq / Hkv;
  for (size_t k = 0; k < bank->desc.size(); ++k) {
    const int nt = tree_tiles(G, bank->desc[k].T);
    const int nqg = query_groups(rows_padded(G, bank->desc[k].T) / kQTile, nt);
    topos[k].splits[0] = 1;
    for (int b = 1; b <= kMaxSplits; ++b)
      topos[k].splits[b] = static_cast<unsigned char>(split_for_bound(b, Hkv * nqg, cus * wg_per_cu(nt)));
  }
}

int32_t launch_attn_device(const entmtp_bank* bank, const DevStep* dev, const DevTopo* topos,
                           const DevAttnShape& sh, const entmtp_bf16* q, const entmtp_bf16* k_tree,
                           const entmtp_bf16* v_tree, entmtp_bf16* k_cache, entmtp_bf16* v_cache,
                           int cap, int Hq, int Hkv, float scale, float rope_theta,
                           entmtp_bf16* out, void* workspace, hipStream_t s) {
  BatchArgs a{};
  a.dev = dev;
  a.topos = topos;
  a.arena = bank->arena;
  a.cus = device_cus();
  a.B = 1;
  a.G = Hq / Hkv;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.cap = cap;
  a.s[0].kc = k_cache;
  a.s[0].vc = v_cache;
  a.scale_log2 = scale * 1.4426950408889634f;
  set_rope(a, rope_theta);
  a.q = q;
  a.kt = k_tree;
  a.vt = v_tree;
  a.out = out;
  // the workspace regions at the bounds workspace_bytes() sizes them with
  const int rows_pad = rows_padded(a.G, sh.T_max);
  const size_t bound = split_bound((cap + sh.T_max + KB - 1) / KB);
  const size_t po = bound * Hkv * rows_pad * HD * sizeof(uint16_t);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  a.part_o = reinterpret_cast<uint16_t*>(ws);
  a.part_ml = reinterpret_cast<float*>(ws + al256(po));
  // one instance per tile count among the bank's trees; those not made for
  // the device's tree leave at once
  for (int nt = 1; nt <= 4; nt *= 2) {
    if (sh.items[nt] == 0) continue;
    a.nt = nt;
    launch_attend(a, sh.items[nt], rope_lds_bytes(sh.D_max, a.theta), s);
    if (int32_t rc = launch_status("tree_attn launch")) return rc;
  }
  hipLaunchKernelGGL(attn_merge_kernel<false>, dim3(sh.merge_blocks), dim3(kMergeThreads), 0, s, a);
  return launch_status("tree_attn merge launch");
}

// Fixed per-sequence ranges of a device-planned batch: each sequence slot
// gets the grid, merge blocks and partial rows of the largest plan any bank
// tree can need at prefix lengths up to cap - T, for either tile count.
struct BatchDevShape {
  int items[5] = {0, 0, 0, 0, 0};   // attend workgroups per sequence, instance with 1 / 4 tiles
  int merge_blocks = 0;             // merge blocks per sequence
  long long part_rows = 0;          // partial rows per sequence
  int D_max = 0;
  size_t need = 0;                  // workspace bytes for B sequences
};

BatchDevShape batch_dev_shape(const entmtp_bank* bank, int B, int Hq, int Hkv, int cap) {
  BatchDevShape sh;
  const int G = Hq / Hkv;
  const int bound = split_bound((cap + KB - 1) / KB);
  int T_max = 0;
  bool any_small = false;
  for (const TopoDesc& td : bank->desc) {
    T_max = td.T > T_max ? td.T : T_max;
    sh.D_max = td.D > sh.D_max ? td.D : sh.D_max;
    any_small = any_small || tree_tiles(G, td.T) == 1;
    // the four-tile instance serves every tree (a batch takes its largest
    // tile count); the one-tile instance only batches of small trees
    const int nqt = rows_padded(G, td.T) / kQTile;
    const int items4 = (Hkv * bound + 7) / 8 * 8 * query_groups(nqt, 4);
    sh.items[4] = items4 > sh.items[4] ? items4 : sh.items[4];
  }
  if (any_small) sh.items[1] = (Hkv * bound + 7) / 8 * 8;
  sh.merge_blocks = (Hkv * G * T_max + kMergeRows - 1) / kMergeRows;
  sh.part_rows = static_cast<long long>(bound) * Hkv * rows_padded(G, T_max);
  const size_t rows = static_cast<size_t>(B) * sh.part_rows;
  sh.need = al256(rows * HD * sizeof(uint16_t)) + al256(rows * 2 * 4);
  return sh;
}

}  // namespace entmtp

// Workspace of entmtp_tree_attn_noalloc, for callers that cannot allocate:
// one array per device, held until the process ends.  Host code never
// passes `scratch` itself to a kernel (in host code the name is a host-side
// stand-in): it takes the device address looked up below.
static __device__ __align__(256) uint8_t scratch[ENTMTP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxScratchDevices] = {};

// Device address of `scratch` on the current device, looked up (with that
// device current) the first time a call runs on it.
int32_t scratch_address(void** out) {
  int dev = -1;
  if (int32_t rc = entmtp::hip_status(hipGetDevice(&dev), "hipGetDevice")) return rc;
  ENTMTP_CHECK_ARG(dev >= 0 && dev < kMaxScratchDevices, ENTMTP_EINVAL,
                   "device %d outside the %d devices the static scratch is tracked for", dev,
                   kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (int32_t rc = entmtp::hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)),
                                        "hipGetSymbolAddress (static scratch)"))
      return rc;
    ENTMTP_CHECK_ARG(p != nullptr, ENTMTP_EHIP, "hipGetSymbolAddress returned NULL for the scratch");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return ENTMTP_OK;
}

}  // namespace

using namespace entmtp;

extern "C" size_t entmtp_tree_attn_workspace(int32_t T, int32_t Hq, int32_t Hkv, int32_t d,
                                             int32_t prefix_len) {
  if (T < 1 || T > ENTMTP_T_MAX || Hq < 1 || Hkv < 1 || Hq % Hkv || d != HD || prefix_len < 0)
    return 0;
  return workspace_bytes(T, Hq, Hkv, prefix_len);
}

extern "C" size_t entmtp_tree_attn_batched_workspace(int32_t B, int32_t T_max, int32_t Hq,
                                                     int32_t Hkv, int32_t d,
                                                     int32_t max_prefix_len) {
  if (B < 1 || B > ENTMTP_B_MAX) return 0;
  return static_cast<size_t>(B) * entmtp_tree_attn_workspace(T_max, Hq, Hkv, d, max_prefix_len);
}

extern "C" int32_t entmtp_tree_attn(const entmtp_bank* bank, int32_t topo, const entmtp_bf16* q,
                                    const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                                    entmtp_bf16* k_cache, entmtp_bf16* v_cache, int32_t cap,
                                    int32_t prefix_len, int32_t Hq, int32_t Hkv, int32_t d,
                                    float scale, float rope_theta, entmtp_bf16* out,
                                    void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  if (int32_t rc = check_sequence(bank, topo, prefix_len, k_cache, v_cache, cap, 0)) return rc;
  if (int32_t rc = check_common(Hq, Hkv, d, scale, rope_theta, q, k_tree, v_tree, out, workspace))
    return rc;
  const int T = bank->desc[topo].T;
  ENTMTP_CHECK_ARG(ws_bytes >= workspace_bytes(T, Hq, Hkv, prefix_len), ENTMTP_ENOSPC,
                   "workspace has %zu bytes, needs %zu", ws_bytes,
                   workspace_bytes(T, Hq, Hkv, prefix_len));
  BatchArgs a;
  const CallShape sh = plan_call(bank, 1, &topo, &prefix_len, &k_cache, &v_cache, cap, Hq, Hkv, a);
  a.scale_log2 = scale * 1.4426950408889634f;
  set_rope(a, rope_theta);
  a.q = q;
  a.kt = k_tree;
  a.vt = v_tree;
  a.out = out;
  return launch_call(a, sh, workspace, static_cast<hipStream_t>(stream));
}

extern "C" int32_t entmtp_tree_attn_noalloc(const entmtp_bank* bank, int32_t topo,
                                            const entmtp_bf16* q, const entmtp_bf16* k_tree,
                                            const entmtp_bf16* v_tree, entmtp_bf16* k_cache,
                                            entmtp_bf16* v_cache, int32_t cap, int32_t prefix_len,
                                            int32_t Hq, int32_t Hkv, int32_t d, float scale,
                                            float rope_theta, entmtp_bf16* out, void* stream) {
  clear_error();
  if (int32_t rc = check_sequence(bank, topo, prefix_len, k_cache, v_cache, cap, 0)) return rc;
  // (the workspace check of check_common is met by the static array)
  if (int32_t rc = check_common(Hq, Hkv, d, scale, rope_theta, q, k_tree, v_tree, out, scratch))
    return rc;
  const int T = bank->desc[topo].T;
  // the bound entmtp_tree_attn_workspace() states covers every plan of the
  // call, so an accepted call stays inside the array
  const size_t need = workspace_bytes(T, Hq, Hkv, prefix_len);
  ENTMTP_CHECK_ARG(need <= ENTMTP_NOALLOC_SCRATCH_BYTES, ENTMTP_ENOSPC,
                   "the call needs %zu bytes of workspace, the static scratch holds %zu", need,
                   static_cast<size_t>(ENTMTP_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  if (int32_t rc = scratch_address(&ws)) return rc;
  BatchArgs a;
  const CallShape sh = plan_call(bank, 1, &topo, &prefix_len, &k_cache, &v_cache, cap, Hq, Hkv, a);
  a.scale_log2 = scale * 1.4426950408889634f;
  set_rope(a, rope_theta);
  a.q = q;
  a.kt = k_tree;
  a.vt = v_tree;
  a.out = out;
  return launch_call(a, sh, ws, static_cast<hipStream_t>(stream));
}

extern "C" int32_t entmtp_tree_attn_batched(
    const entmtp_bank* bank, int32_t B, const int32_t* topo, const int32_t* prefix_len,
    const entmtp_bf16* q, const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
    entmtp_bf16* const* k_caches, entmtp_bf16* const* v_caches, int32_t cap, int32_t Hq,
    int32_t Hkv, int32_t d, float scale, float rope_theta, entmtp_bf16* out, void* workspace,
    size_t ws_bytes, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 1 && B <= ENTMTP_B_MAX, ENTMTP_EINVAL, "B = %d outside [1, %d]", B,
                   ENTMTP_B_MAX);
  ENTMTP_CHECK_ARG(topo && prefix_len && k_caches && v_caches, ENTMTP_EINVAL,
                   "topo, prefix_len, k_caches and v_caches must be non-NULL host arrays");
  for (int b = 0; b < B; ++b)
    if (int32_t rc = check_sequence(bank, topo[b], prefix_len[b], k_caches[b], v_caches[b], cap, b))
      return rc;
  if (int32_t rc = check_common(Hq, Hkv, d, scale, rope_theta, q, k_tree, v_tree, out, workspace))
    return rc;
  BatchArgs a;
  const CallShape sh = plan_call(bank, B, topo, prefix_len, k_caches, v_caches, cap, Hq, Hkv, a);
  ENTMTP_CHECK_ARG(ws_bytes >= sh.need, ENTMTP_ENOSPC, "workspace has %zu bytes, needs %zu",
                   ws_bytes, sh.need);
  a.scale_log2 = scale * 1.4426950408889634f;
  set_rope(a, rope_theta);
  a.q = q;
  a.kt = k_tree;
  a.vt = v_tree;
  a.out = out;
  return launch_call(a, sh, workspace, static_cast<hipStream_t>(stream));
}

extern "C" size_t entmtp_tree_attn_batched_device_workspace(const entmtp_bank* bank, int32_t B,
                                                            int32_t Hq, int32_t Hkv, int32_t d,
                                                            int32_t cap) {
  if (!bank || bank->desc.empty() || B < 1 || B > ENTMTP_B_MAX || Hq < 1 || Hkv < 1 ||
      Hq % Hkv || d != HD || cap < 1)
    return 0;
  return batch_dev_shape(bank, B, Hq, Hkv, cap).need;
}

extern "C" int32_t entmtp_tree_attn_batched_device(
    const entmtp_bank* bank, int32_t B, const int32_t* topo, const int32_t* prefix_len,
    const int32_t* row_off, int32_t rows_cap, const entmtp_bf16* q, const entmtp_bf16* k_tree,
    const entmtp_bf16* v_tree, entmtp_bf16* const* k_caches, entmtp_bf16* const* v_caches,
    int32_t cap, int32_t Hq, int32_t Hkv, int32_t d, float scale, float rope_theta,
    entmtp_bf16* out, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  ENTMTP_CHECK_ARG(B >= 1 && B <= ENTMTP_B_MAX, ENTMTP_EINVAL, "B = %d outside [1, %d]", B,
                   ENTMTP_B_MAX);
  if (int32_t rc = check_device_bank(bank, 0)) return rc;
  ENTMTP_CHECK_ARG(static_cast<int>(bank->desc.size()) <= kMaxTreesArg, ENTMTP_ERANGE,
                   "a device-planned batch names at most %d bank trees (bank has %zu)",
                   kMaxTreesArg, bank->desc.size());
  ENTMTP_CHECK_ARG(topo && prefix_len && row_off, ENTMTP_EINVAL,
                   "topo, prefix_len and row_off must be non-NULL device arrays");
  ENTMTP_CHECK_ARG(k_caches && v_caches, ENTMTP_EINVAL,
                   "k_caches and v_caches must be non-NULL host arrays");
  ENTMTP_CHECK_ARG(rows_cap >= 1, ENTMTP_EINVAL, "rows_cap = %d < 1", rows_cap);
  ENTMTP_CHECK_ARG(cap >= 1, ENTMTP_EINVAL, "cap = %d < 1", cap);
  for (int b = 0; b < B; ++b)
    ENTMTP_CHECK_ARG(k_caches[b] && v_caches[b] && aligned16(k_caches[b]) && aligned16(v_caches[b]),
                     ENTMTP_EINVAL, "sequence %d: caches must be non-NULL and 16-byte aligned", b);
  if (int32_t rc = check_common(Hq, Hkv, d, scale, rope_theta, q, k_tree, v_tree, out, workspace))
    return rc;
  const BatchDevShape sh = batch_dev_shape(bank, B, Hq, Hkv, cap);
  ENTMTP_CHECK_ARG(ws_bytes >= sh.need, ENTMTP_ENOSPC, "workspace has %zu bytes, needs %zu",
                   ws_bytes, sh.need);
  BatchArgs a{};
  a.topo_dev = topo;
  a.len_dev = prefix_len;
  a.row_off_dev = row_off;
  a.rows_cap = rows_cap;
  a.n_trees = static_cast<int>(bank->desc.size());
  for (int k = 0; k < a.n_trees; ++k) {
    const TopoDesc& td = bank->desc[k];
    ENTMTP_CHECK_ARG(td.off_mask <= INT32_MAX && td.off_depth <= INT32_MAX, ENTMTP_ERANGE,
                     "bank arena offsets past 2 GiB");
    a.trees[k] = TreeHdr{td.T, td.D, static_cast<int>(td.off_mask), static_cast<int>(td.off_depth)};
  }
  a.arena = bank->arena;
  a.cus = device_cus();
  a.B = B;
  a.G = Hq / Hkv;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.cap = cap;
  a.scale_log2 = scale * 1.4426950408889634f;
  set_rope(a, rope_theta);
  a.q = q;
  a.kt = k_tree;
  a.vt = v_tree;
  a.out = out;
  const size_t rows = static_cast<size_t>(B) * sh.part_rows;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  a.part_o = reinterpret_cast<uint16_t*>(ws);
  a.part_ml = reinterpret_cast<float*>(ws + al256(rows * HD * sizeof(uint16_t)));
  for (int b = 0; b < B; ++b) {
    a.s[b].kc = k_caches[b];
    a.s[b].vc = v_caches[b];
    a.s[b].merge0 = b * sh.merge_blocks;
    a.s[b].part_off = b * sh.part_rows;
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  // one instance per tile count; a batch's workgroups in the other leave at once
  for (int nt = 1; nt <= 4; nt *= 4) {
    if (sh.items[nt] == 0) continue;
    a.nt = nt;
    for (int b = 0; b < B; ++b) a.s[b].item0 = b * sh.items[nt];
    launch_attend<true>(a, B * sh.items[nt], rope_lds_bytes(sh.D_max, a.theta), s);
    if (int32_t rc = launch_status("tree_attn (device-planned batch) launch")) return rc;
  }
  hipLaunchKernelGGL(attn_merge_kernel<true>, dim3(B * sh.merge_blocks), dim3(kMergeThreads), 0, s, a);
  return launch_status("tree_attn (device-planned batch) merge launch");
}
