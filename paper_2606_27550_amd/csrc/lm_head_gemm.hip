// LM head over many rows: the verification logits of §2.3 for a batch of
// trees verified together (up to hundreds of rows), as a tiled MFMA
// contraction.
//
// With hundreds of rows the product logits = X W^T is no longer a skinny
// stream: at 544 rows and a 128256-entry vocabulary it holds 571 GFLOP for
// 1.05 GB of W, so it is bound by the matrix cores, not HBM.  The streaming
// kernels take at most 128 rows per pass and stage W through registers of
// one wave per 16 rows; this kernel gives a workgroup a 256-row vocabulary
// block (four of the streaming grid's slices) and 128 rows of X, shared
// through LDS, so each LDS byte feeds 64 to 128 products:
//  * eight waves in a 4 x 2 grid over the 256 x 128 output tile (two per
//    SIMD, so one issues products while the other waits), each accumulating
//    a 64 x 64 sub-tile with v_mfma_f32_16x16x32_bf16 (128-row blocks: four
//    waves, 2 x 2);
//  * K advances in stages of 64: each wave loads its share of a stage's W
//    and X rows into VGPRs (8 rows x 128 bytes per instruction) two stages
//    ahead of storing them into one of three LDS slots, two stages ahead of
//    their use (direct global->LDS copies measured at a third of the rate
//    this tile consumes; 16 rows x 64 bytes per instruction at two thirds);
//  * within a 128-byte row the eight 16-byte chunks are stored XOR-swizzled
//    by the row's place in its 16-row group, so the MFMA fragment reads
//    (16 rows, one chunk) spread over all LDS banks;
//  * the stores, loads and fragment reads of a stage are interleaved one by
//    one with its products, and a k-step's fragments are read during the
//    previous k-step; one LDS wait and one barrier per stage;
//  * the passes of one vocabulary block run on one XCD (dispatch is
//    round-robin), so W fetched by one pass is an L2 hit for the others;
//  * each wave runs a form of the tile specialised to the number of its
//    16-row X blocks that hold rows of the batch, so the last pass of a
//    ragged batch (16 of 128 rows at 400) skips the padding's products;
//  * with statistics the epilogue reduces each row's accumulators over the
//    block into one partial (the streaming kernels' layout: the block's
//    partial in its first slice, neutral partials in the other three), so
//    the statistics merge is unchanged.
// Hidden sizes 4096 and 5120 (the stage count is a template parameter).
#include <type_traits>

#include "common.hpp"
#include "stats.hpp"
#include "stream_pipe.hpp"

namespace entmtp {
namespace {

constexpr int kGemmBN = 128;        // rows of X per pass
constexpr int kGemmBK = 64;         // k per stage: two MFMA k-steps, 128-byte rows
constexpr int kGemmMinRows = 128;   // the streaming kernels' largest pass
constexpr int kGemmSlots = 3;       // LDS stages: multiplied, read, written
constexpr int kGemmD = 2;           // stages of loads held in VGPRs ahead of their store

// BM vocabulary rows per block: BM / 64 of the streaming grid's slices (at
// most 64 rows each), 256 when the vocabulary gives every CU a block (128256
// entries: 501 blocks), else 128 (32000: 250).
// NW waves: NW / 2 along the vocabulary rows, two along the rows of X.
template <int BM, int BN, int NW>
struct GemmShape {
  static constexpr int THREADS = 64 * NW;
  static constexpr int WMW = NW / 2;              // waves along M
  static constexpr int SLICES = BM / 64;
  static constexpr int ROWB = kGemmBK * 2;        // bytes of a row per stage
  static constexpr int CH = ROWB / 16;            // 16-byte chunks per row
  static constexpr int RPI = 64 / CH;             // rows per load instruction (8)
  static constexpr int A_BYTES = BM * ROWB;       // W block
  static constexpr int B_BYTES = BN * ROWB;       // X block
  static constexpr int SLOT = A_BYTES + B_BYTES;
  static constexpr int AI = BM / RPI / NW;        // W loads per wave per stage
  static constexpr int BI = BN / RPI / NW;        // X loads per wave per stage
  static constexpr int LI = AI + BI;
  static constexpr int WM = BM / WMW, WN = BN / 2;   // wave sub-tile
  static constexpr int MI = WM / 16, NI = WN / 16;
  static constexpr int NF = MI + NI;              // fragments per k-step
  // Accumulators in AGPRs when a wave's 128 x 64 sub-tile needs 128 of them
  // beside ~220 VGPRs (one wave per SIMD); with two waves per SIMD the
  // compiler halves the 256-register budget between the two files once
  // AGPRs are used, so 64 x 64 sub-tiles keep theirs in VGPRs.
  static constexpr bool ACC_AGPR = NW == 4;
  static_assert(BN % (NW * RPI) == 0 && AI % 2 == 0 && BI % 2 == 0, "loads split evenly");
  static_assert(kGemmSlots * SLOT <= 160 * 1024, "slots fit in LDS");
};

// Slot of 16-byte chunk c of row r (eight chunks per row) is c ^ swz(r).  A
// fragment read takes one chunk of 16 consecutive rows (128-byte rows).  The
// LDS serves a 16-byte read for 32 lanes per cycle (512 bytes: lanes of two
// chunk columns over 16 rows), which conflicts unless the 32 addresses fall
// in distinct 16-byte bank groups mod 512 bytes: rows r, r + 4, r + 8, r + 12
// must differ in swz >> 1.  swz also keeps 16- and 8-lane groups apart (rows
// of one parity, and rows 0..7 / 8..15, distinct), found by a search over
// XOR swizzles; the bank-conflict counter reads 0.2 % of the simpler
// (r & 7) ^ (r >> 3 & 1), which conflicted in the 32-lane groups.
__device__ __forceinline__ int chunk_swz(int r) { return ((r >> 1) & 3) | (((r ^ (r >> 3)) & 1) << 2); }

// s_waitcnt lgkmcnt(N) alone (vmcnt and expcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_lds_but() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  __builtin_amdgcn_s_waitcnt(0xC07F | (N << 8));
}
__device__ __forceinline__ void wait_lds() { wait_lds_but<0>(); }

// True when each of h groups of m products (split as evenly as integer
// division gives) has a product ahead of each of its accesses: a store, a
// load and its share of f fragment reads.
constexpr bool gemm_groups_fit(int m, int h, int f) {
  for (int g = 0; g < h; ++g)
    if (2 + f * (g + 1) / h - f * g / h > m * (g + 1) / h - m * g / h) return false;
  return true;
}

// Waits out the latency of the last MFMAs before their accumulators are
// read (32 wait states: the longest 16x16x32 result latency is 16 passes of
// four cycles, of which the issue of the following instructions covers the
// rest).
__device__ __forceinline__ void mfma_drain() {
  asm volatile("s_nop 15\n\ts_nop 15" ::: "memory");
}

// The workgroup's tile (vocabulary rows [r0, r1), batch rows from j0),
// with NA = the number of the wave's 16-row X blocks that hold rows of the
// batch: the last pass of a ragged batch leaves out the products of the
// others (loads, stores, fragment reads and barriers are the same in every
// form, so the waves of a workgroup stay in step).
template <int BM, int BN, int NW, int NST, bool STATS, int NA>
__device__ __forceinline__ void gemm_tile(
    uint8_t* __restrict__ ring, const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
    float* __restrict__ logits, int T, int hid, int V, int G, float inv_temp,
    StatPart* __restrict__ part, int grp, int j0, int r0, int r1) {
  using Sh = GemmShape<BM, BN, NW>;
  constexpr int kSlices = Sh::SLICES;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const StatPart empty{-INFINITY, 0.f, 0.f, 0x7fffffff};
  // load instruction q of a wave covers rows (wave * n + q) * 8 .. + 7 of
  // the block (n = AI for W, BI for X); lane l takes chunk l % 8 of row l / 8
  // and stores it at slot (l % 8) ^ swz(row).  W rows past the block load
  // the next block's rows (or the last row of W), X rows past T the pass's
  // first row: in bounds, and never stored.
  const int lrow = lane >> 3, lch = lane & 7;
  uint32_t src[Sh::LI];   // byte offsets from W (q < AI) or X
#pragma unroll
  for (int q = 0; q < Sh::AI; ++q) {
    const int row = min(r0 + (wave * Sh::AI + q) * Sh::RPI + lrow, V - 1);
    src[q] = (static_cast<uint32_t>(row) * hid + 8 * lch) * 2u;
  }
#pragma unroll
  for (int q = 0; q < Sh::BI; ++q) {
    const int rr = (wave * Sh::BI + q) * Sh::RPI + lrow;
    const int node = j0 + rr < T ? j0 + rr : j0;
    src[Sh::AI + q] = (static_cast<uint32_t>(node) * hid + 8 * lch) * 2u;
  }
  // LDS byte offset of the lane's chunk for load q (rows of one instruction
  // are 8 apart within the block, so the swizzle depends on q's parity)
  auto dst_of = [&](int q) {
    const int rr = q < Sh::AI ? (wave * Sh::AI + q) * Sh::RPI + lrow
                              : (wave * Sh::BI + q - Sh::AI) * Sh::RPI + lrow;
    return (q < Sh::AI ? 0 : Sh::A_BYTES) + rr * Sh::ROWB + ((lch ^ chunk_swz(rr)) << 4);
  };
  // blocks walk K in rotated order, so that CUs do not all stream the same
  // column band of W at once
  const int rot = static_cast<int>((static_cast<unsigned>(grp) * 7u) % static_cast<unsigned>(NST));
  const uint8_t* const Wb = reinterpret_cast<const uint8_t*>(W);
  const uint8_t* const Xb = reinterpret_cast<const uint8_t*>(X);
  u32x4 pre[kGemmD][Sh::LI];
  // load q of stage `stage` (clamped to the last stage)
  auto load_one = [&](u32x4& r, int q, int stage) {
    int ks = (stage < NST ? stage : NST - 1) + rot;
    ks = ks >= NST ? ks - NST : ks;
    const uint32_t off = src[q] + static_cast<uint32_t>(ks * Sh::ROWB);
    // W is streamed once: keep it out of the caches' way; X is re-read
    if (q < Sh::AI)
      r = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Wb + off));
    else
      r = *reinterpret_cast<const u32x4*>(Xb + off);
  };

  const int lr = lane & 15, lg = lane >> 4;
  const int wm = wave % Sh::WMW, wn = wave / Sh::WMW;
  // fragment f of k-step j: W block f (f < MI) rows wm*WM + 16f + lr, or X
  // block f - MI rows wn*WN + 16(f - MI) + lr; chunk 4j + lg
  auto read_one = [&](bf16x8& out, const uint8_t* slot, int j, int f) {
    const int row = f < Sh::MI ? wm * Sh::WM + 16 * f + lr : wn * Sh::WN + 16 * (f - Sh::MI) + lr;
    const int off = (f < Sh::MI ? 0 : Sh::A_BYTES) + row * Sh::ROWB + (((4 * j + lg) ^ chunk_swz(lr)) << 4);
    out = as_bf16x8(*reinterpret_cast<const u32x4*>(slot + off));
  };

  f32x4 acc[Sh::MI][Sh::NI];
#pragma unroll
  for (int mi = 0; mi < Sh::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < Sh::NI; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 frag[2][Sh::NF];
  // The products accumulate in place (AGPRs or VGPRs), as inline assembly:
  // with the builtin the compiler renamed the accumulators from one step to
  // the next and spent a move per accumulator register per loop trip
  // undoing it.  The "memory" clobber keeps the step's loads, stores and
  // fragment reads where the source puts them among the products.  Nothing
  // reads an accumulator between products; mfma_drain() covers the window
  // before the epilogue reads them.
  auto mfma_one = [&](int buf, int i) {
    const int mi = i / Sh::NI, ni = i % Sh::NI;
    if (ni >= NA) return;   // an X block wholly past the batch
    if constexpr (Sh::ACC_AGPR)
      asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                   : "+a"(acc[mi][ni])
                   : "v"(frag[buf][mi]), "v"(frag[buf][Sh::MI + ni])
                   : "memory");
    else
      asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                   : "+v"(acc[mi][ni])
                   : "v"(frag[buf][mi]), "v"(frag[buf][Sh::MI + ni])
                   : "memory");
  };
  // An empty assembly statement that takes and returns every accumulator.
  // mfma_drain() orders memory accesses only: without this the compiler may
  // schedule arithmetic on the accumulators (the statistics epilogue) ahead of
  // the drain, into the last products' latency, or sink their zeroing past it
  // towards the first products.  Pinned right after the zeroing and right
  // after the final drain, they cross neither (the assembly statements keep
  // their order).
  auto pin_acc = [&]() {
#pragma unroll
    for (int mi = 0; mi < Sh::MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < Sh::NI; ++ni) {
        if constexpr (Sh::ACC_AGPR)
          asm volatile("" : "+a"(acc[mi][ni]));
        else
          asm volatile("" : "+v"(acc[mi][ni]));
      }
  };
  // the fragments in the order the products need them: X blocks (every
  // product of the first W block uses one), then W blocks
  auto frag_at = [&](int n) { return n < Sh::NI ? Sh::MI + n : n - Sh::NI; };

  // Stage s is loaded into pre[s % D] at step s - 2 - D (the prologue for
  // the first ones), stored into slot s % 3 at step s - 2, its first k-step's
  // fragments read during step s - 1, its second's during step s, and it is
  // multiplied at step s.  A slot is overwritten two steps after its last
  // fragments were read, behind a barrier.  Loads past the last stage
  // re-load it.
#pragma unroll
  for (int k = 0; k < kGemmD; ++k)
#pragma unroll
    for (int q = 0; q < Sh::LI; ++q) load_one(pre[k][q], q, k);
#pragma unroll
  for (int k = 0; k < 2; ++k)
#pragma unroll
    for (int q = 0; q < Sh::LI; ++q) {
      *reinterpret_cast<u32x4*>(ring + k * Sh::SLOT + dst_of(q)) = pre[k % kGemmD][q];
      load_one(pre[k % kGemmD][q], q, kGemmD + k);
    }
  wait_lds();
  stage_barrier();
#pragma unroll
  for (int n = 0; n < Sh::NF; ++n) read_one(frag[0][frag_at(n)], ring, 0, frag_at(n));
  pin_acc();
  mfma_drain();   // the accumulators' zeroing precedes their first product

  // Step c, K = c mod 6 (slot and load set depend on K only).  A k-step's
  // products run in LI / 2 groups; after the products of group g, one at a
  // time: a store of stage c + 2 (half of them per k-step), the load of
  // stage c + 2 + D that refills its registers, and the group's share of the
  // fragments of the next k-step (stage c's second in k-step 0, stage c + 1's
  // first in k-step 1).  Issued in one burst the LDS accesses filled the LDS
  // queue and the wave stalled there with the matrix pipe idle.  The last
  // group's reads follow the step's last store, so lgkmcnt(kTailReads) at the
  // end means the step's stores have landed.
  constexpr int kMma = Sh::MI * Sh::NI;
  constexpr int kHalf = Sh::LI / 2;
  constexpr int kTailReads = Sh::NF - Sh::NF * (kHalf - 1) / kHalf;
  static_assert(gemm_groups_fit(kMma, kHalf, Sh::NF) && kTailReads < 16,
                "every group's accesses follow products of its own");
  auto kstep = [&](int j, uint8_t* wslot, u32x4 (&pr)[Sh::LI], const uint8_t* rslot, int rj,
                   int c) {
#pragma unroll
    for (int g = 0; g < kHalf; ++g) {
      const int q = j * kHalf + g;
      const int lo = kMma * g / kHalf, hi = kMma * (g + 1) / kHalf;   // this group's products
      const int f0 = Sh::NF * g / kHalf, f1 = Sh::NF * (g + 1) / kHalf;   // and fragments
      mfma_one(j, lo);
      *reinterpret_cast<u32x4*>(wslot + dst_of(q)) = pr[q];
      mfma_one(j, lo + 1);
      load_one(pr[q], q, c + 2 + kGemmD);
#pragma unroll
      for (int f = f0; f < f1; ++f) {
        mfma_one(j, lo + 2 + f - f0);
        read_one(frag[j ^ 1][frag_at(f)], rslot, rj, frag_at(f));
      }
#pragma unroll
      for (int i = lo + 2 + f1 - f0; i < hi; ++i) mfma_one(j, i);
    }
  };
  auto step = [&](auto kc, int c) {
    constexpr int K = decltype(kc)::value;
    uint8_t* wslot = ring + ((K + 2) % kGemmSlots) * Sh::SLOT;
    u32x4 (&pr)[Sh::LI] = pre[(K + 2) % kGemmD];
    kstep(0, wslot, pr, ring + (K % kGemmSlots) * Sh::SLOT, 1, c);
    kstep(1, wslot, pr, ring + ((K + 1) % kGemmSlots) * Sh::SLOT, 0, c);
    wait_lds_but<kTailReads>();
    stage_barrier();
  };
  static_assert(6 % kGemmD == 0, "six steps return slots and load sets to their start");
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  using I4 = std::integral_constant<int, 4>;
  using I5 = std::integral_constant<int, 5>;
  constexpr int kRounds = NST / 6;
  for (int c = 0; c < 6 * kRounds; c += 6) {
    step(I0{}, c);
    step(I1{}, c + 1);
    step(I2{}, c + 2);
    step(I3{}, c + 3);
    step(I4{}, c + 4);
    step(I5{}, c + 5);
  }
  constexpr int kTail = NST - 6 * kRounds;
  if constexpr (kTail > 0) step(I0{}, 6 * kRounds);
  if constexpr (kTail > 1) step(I1{}, 6 * kRounds + 1);
  if constexpr (kTail > 2) step(I2{}, 6 * kRounds + 2);
  if constexpr (kTail > 3) step(I3{}, 6 * kRounds + 3);
  if constexpr (kTail > 4) step(I4{}, 6 * kRounds + 4);
  mfma_drain();
  pin_acc();

  const int vbase = r0 + wm * Sh::WM + 4 * lg;   // first of the lane's rows in block mi = 0
  if (logits) {
    const bool vec_ok = (V & 3) == 0;
#pragma unroll
    for (int mi = 0; mi < Sh::MI; ++mi) {
      const int v = vbase + 16 * mi;
      // one block row at a time: the scheduler would otherwise pull every
      // accumulator out of the AGPRs at once and spill
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ni = 0; ni < Sh::NI; ++ni) {
        const int node = j0 + wn * Sh::WN + 16 * ni + lr;
        if (node >= T) continue;
        float* dst = logits + static_cast<size_t>(node) * V + v;
        if (vec_ok && v + 3 < r1) {
          *reinterpret_cast<f32x4*>(dst) = acc[mi][ni];
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (v + r < r1) dst[r] = acc[mi][ni][r];
        }
      }
    }
  }
  if constexpr (STATS) {
    // per row: the wave's partial over its WM vocabulary rows (lane, then
    // the four lane groups), then the row's NW / 2 waves in LDS.  A lane
    // visits its rows in increasing order, so within the lane a strictly
    // larger value is the only update the lowest-index rule needs.  The
    // sums run in base 2 (one hardware exponential per logit): with
    // y2 = log2(e) (inv_temp z - my), Z = sum 2^y2 and S = ln 2 sum y2 2^y2.
    constexpr float kLog2e = 1.44269504088896341f, kLn2 = 0.69314718055994531f;
    const float it2 = inv_temp * kLog2e;
    const bool full = r1 - r0 == BM;   // every row of the block is a vocabulary row
    StatPart* wpart = reinterpret_cast<StatPart*>(ring);   // [WMW][BN]
#pragma unroll
    for (int ni = 0; ni < Sh::NI; ++ni) {
      __builtin_amdgcn_sched_barrier(0);   // one node column at a time (as above)
      StatPart p = empty;
#pragma unroll
      for (int mi = 0; mi < Sh::MI; ++mi)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int v = vbase + 16 * mi + r;
          if ((full || v < r1) && acc[mi][ni][r] > p.zmax) {
            p.zmax = acc[mi][ni][r];
            p.idx = v;
          }
        }
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1)
        take_max(p.zmax, p.idx, __shfl_xor(p.zmax, off, 64), __shfl_xor(p.idx, off, 64));
      if (p.zmax != -INFINITY) {
        const float my2 = p.zmax * it2;
        float Z = 0.f, S2 = 0.f;
#pragma unroll
        for (int mi = 0; mi < Sh::MI; ++mi)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if (full || vbase + 16 * mi + r < r1) {
              const float y2 = fmaf(acc[mi][ni][r], it2, -my2);
              const float e = __builtin_amdgcn_exp2f(y2);
              Z += e;
              S2 = fmaf(y2, e, S2);
            }
          }
        p.Z = Z;
        p.S = S2 * kLn2;
      }
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        p.Z += __shfl_xor(p.Z, off, 64);
        p.S += __shfl_xor(p.S, off, 64);
      }
      if (lg == 0) wpart[wm * BN + wn * Sh::WN + 16 * ni + lr] = p;
    }
    __syncthreads();
    for (int c = tid; c < BN; c += Sh::THREADS) {
      if (j0 + c >= T) continue;
      StatPart q = wpart[c];
#pragma unroll
      for (int w = 1; w < Sh::WMW; ++w) part_merge(q, wpart[w * BN + c], inv_temp);
      StatPart* dst = part + static_cast<size_t>(j0 + c) * G + kSlices * grp;
      dst[0] = q;
#pragma unroll
      for (int u = 1; u < kSlices; ++u)
        if (kSlices * grp + u < G) dst[u] = empty;
    }
  }
}

template <int BM, int BN, int NW, int NST, bool STATS>
__global__ __launch_bounds__(64 * NW) void lm_head_gemm_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, float* __restrict__ logits,
    int T, int hid, int V, int G, float inv_temp, StatPart* __restrict__ part) {
  using Sh = GemmShape<BM, BN, NW>;
  constexpr int kSlices = Sh::SLICES;
  __shared__ __attribute__((aligned(16))) uint8_t ring[kGemmSlots * Sh::SLOT];

  // 1-D grid over (block group, pass, XCD): the passes of one vocabulary
  // block are consecutive workgroups of one XCD
  const int groups = (G + kSlices - 1) / kSlices;
  const int passes = (T + BN - 1) / BN;
  const int bid = blockIdx.x, r8 = bid >> 3;
  const int pass = r8 % passes, grp = (r8 / passes) * 8 + (bid & 7);
  if (grp >= groups) return;
  const int j0 = pass * BN;
  const int r0 = slice_begin(kSlices * grp, G, V);
  const int r1 = slice_begin(kSlices * grp + kSlices, G, V);
  const int tid = threadIdx.x, wave = tid >> 6;
  const StatPart empty{-INFINITY, 0.f, 0.f, 0x7fffffff};
  if (r0 >= r1) {   // empty block (tiny V): neutral partials only
    if constexpr (STATS)
      for (int c = tid; c < BN; c += Sh::THREADS)
        if (j0 + c < T)
          for (int u = 0; u < kSlices && kSlices * grp + u < G; ++u)
            part[static_cast<size_t>(j0 + c) * G + kSlices * grp + u] = empty;
    return;
  }
  // live X blocks of the wave (wave-uniform)
  const int na = __builtin_amdgcn_readfirstlane(
      min(max((T - j0 - (wave / Sh::WMW) * Sh::WN + 15) / 16, 0), Sh::NI));
  static_assert(Sh::NI == 4, "one form per live X block count");
  switch (na) {
    case 0:
      gemm_tile<BM, BN, NW, NST, STATS, 0>(ring, X, W, logits, T, hid, V, G, inv_temp, part, grp, j0, r0, r1);
      break;
    case 1:
      gemm_tile<BM, BN, NW, NST, STATS, 1>(ring, X, W, logits, T, hid, V, G, inv_temp, part, grp, j0, r0, r1);
      break;
    case 2:
      gemm_tile<BM, BN, NW, NST, STATS, 2>(ring, X, W, logits, T, hid, V, G, inv_temp, part, grp, j0, r0, r1);
      break;
    case 3:
      gemm_tile<BM, BN, NW, NST, STATS, 3>(ring, X, W, logits, T, hid, V, G, inv_temp, part, grp, j0, r0, r1);
      break;
    default:
      gemm_tile<BM, BN, NW, NST, STATS, 4>(ring, X, W, logits, T, hid, V, G, inv_temp, part, grp, j0, r0, r1);
  }
}

template <int BM, int NW, int NST, bool STATS>
int32_t launch_gemm(const uint16_t* X, const uint16_t* W, float* logits, int T, int hid, int V,
                    int G, float inv_temp, StatPart* part, hipStream_t s) {
  constexpr int kSlices = BM / 64;
  const int groups = (G + kSlices - 1) / kSlices;
  const int passes = (T + kGemmBN - 1) / kGemmBN;
  const int blocks = (groups + 7) / 8 * passes * 8;
  hipLaunchKernelGGL((lm_head_gemm_kernel<BM, kGemmBN, NW, NST, STATS>), dim3(blocks),
                     dim3(64 * NW), 0, s, X, W, logits, T, hid, V, G, inv_temp, part);
  return launch_status("verify_logits (tiled) launch");
}

// 256-row blocks: eight waves (4 x 2, two per SIMD) measured 2-3 % faster
// than four (2 x 2) at 90-544 rows.
constexpr int kWideWaves = 8;

template <int NST>
int32_t launch_gemm_bm(bool wide, const uint16_t* X, const uint16_t* W, float* logits, int T,
                       int hid, int V, int G, float inv_temp, StatPart* part, hipStream_t s) {
  if (wide)
    return part ? launch_gemm<256, kWideWaves, NST, true>(X, W, logits, T, hid, V, G, inv_temp, part, s)
                : launch_gemm<256, kWideWaves, NST, false>(X, W, logits, T, hid, V, G, inv_temp, nullptr, s);
  return part ? launch_gemm<128, 4, NST, true>(X, W, logits, T, hid, V, G, inv_temp, part, s)
              : launch_gemm<128, 4, NST, false>(X, W, logits, T, hid, V, G, inv_temp, nullptr, s);
}

}  // namespace

bool lm_gemm_takes(int T, int hid, int G, int cus) {
  if ((hid != 64 * kGemmBK && hid != 80 * kGemmBK) || G % 4 != 0) return false;
  // more than one streaming pass of 128 rows, or more than 64 rows and a
  // block per CU
  return T > kGemmMinRows || (T > kGemmMinRows / 2 && G / 2 >= cus);
}

int32_t launch_lm_gemm(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, float* logits, int T,
                       int hid, int V, int G, float inv_temp, void* partials, int cus,
                       hipStream_t s) {
  const auto* X = reinterpret_cast<const uint16_t*>(hidden);
  const auto* W = reinterpret_cast<const uint16_t*>(w_lm);
  auto* part = static_cast<StatPart*>(partials);
  const bool wide = G / 4 >= cus;   // 256-row blocks still give every CU one
  if (hid == 64 * kGemmBK) return launch_gemm_bm<64>(wide, X, W, logits, T, hid, V, G, inv_temp, part, s);
  return launch_gemm_bm<80>(wide, X, W, logits, T, hid, V, G, inv_temp, part, s);
}

}  // namespace entmtp
