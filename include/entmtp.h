/*
 * entmtp.h -- C ABI of the EntMTP tree-verification hot path on AMD Instinct
 * MI355X (gfx950).
 *
 * One decode step of a multi-token-prediction decoder verifies a draft tree in
 * a single sparse forward pass (paper §2.3), then keeps the longest accepted
 * root-to-node path and updates the KV cache (§3.2 loop: proposal -> tree
 * decoding -> verification -> KV-cache update).  The scheduler of §4 picks the
 * tree for every step from a precompiled bank, so that switching trees is an
 * index change with no rebuild (§4 "Cost").  This library implements that
 * pass:
 *
 *   entmtp_bank_build     per-tree buffers (mask, position offsets, gather rows)
 *   entmtp_tree_attn      tree-masked attention over prefix KV + the tree
 *   entmtp_verify_logits  LM-head logits of the tree's final hidden states
 *   entmtp_logit_stats    per-node entropy, top-1 probability and argmax
 *   entmtp_accept         longest accepted path, bonus token
 *   entmtp_kv_compact     KV-cache compaction of the accepted path
 *
 * Conventions shared by every call:
 *   - Tensor pointers are DEVICE pointers owned by the caller unless the
 *     argument is documented as host memory.  bf16 tensors are passed as
 *     uint16_t bit patterns (entmtp_bf16).  All layouts are dense row-major.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls that
 *     launch work are asynchronous on `stream` and never synchronise it,
 *     except entmtp_bank_build (see there).
 *   - Every argument is validated on the host before anything is launched,
 *     so a call that returns an error has launched nothing.
 *   - Return value: ENTMTP_OK (0) or a negative status; the message of the
 *     last error of the calling thread is returned by entmtp_last_error().
 *   - Asynchronous device faults surface at a later synchronisation of the
 *     stream, not as a return code of the call that launched the kernel.
 */
#ifndef ENTMTP_H
#define ENTMTP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ENTMTP_OK       0
#define ENTMTP_EINVAL  (-1)  /* null pointer, bad size, unsupported shape, topo out of range */
#define ENTMTP_ETREE   (-2)  /* malformed tree: parent[0] != -1 or parent[i] not in [0, i) */
#define ENTMTP_ERANGE  (-3)  /* T > ENTMTP_T_MAX, depth > ENTMTP_D_MAX, cap < L+T, Hq % Hkv */
#define ENTMTP_ENOSPC  (-4)  /* arena or workspace smaller than required */
#define ENTMTP_EHIP    (-5)  /* HIP runtime or launch error (message kept) */
#define ENTMTP_ETIMEDOUT (-6)  /* entmtp_step_wait: no result within the time limit */

#define ENTMTP_T_MAX      256  /* nodes per tree, root included */
#define ENTMTP_D_MAX      31   /* deepest node (root = depth 0) */
#define ENTMTP_MASK_WORDS 8    /* uint32 words per mask row (ENTMTP_T_MAX / 32) */
#define ENTMTP_HEAD_DIM   128  /* the head dimension the attention kernels are built for */
#define ENTMTP_B_MAX      16   /* sequences per batched call */

typedef uint16_t entmtp_bf16;
typedef struct entmtp_bank entmtp_bank;

/* Message of the calling thread's last error ("" if none).  Never NULL. */
const char* entmtp_last_error(void);

/* Library version string. */
const char* entmtp_version(void);

/* ------------------------------------------------------------------------ */
/* TopologyBank (§2.3: trees ship precomputed attention masks, position       */
/* offsets and gather indices; §4 "Cost": one buffer set per tree, switching  */
/* trees is a pointer swap).                                                  */
/* ------------------------------------------------------------------------ */

/*
 * Build the bank of `n_trees` draft trees.
 *
 *   parents_host   host int32[sum(sizes)]: the trees' parent arrays back to
 *                  back.  Node 0 of each tree is its root (parent -1); every
 *                  other node's parent is an earlier node of the same tree.
 *   sizes_host     host int32[n_trees]: node count T of each tree (root
 *                  included), 1 <= T <= ENTMTP_T_MAX.
 *   arena          device buffer that will hold the bank, or NULL.
 *   arena_bytes    size of `arena`.
 *   arena_needed   host out (optional): bytes the arena must have.
 *   stream         stream of the upload.
 *   out            host out: the bank handle (owned by the library, free with
 *                  entmtp_bank_destroy).  May be NULL when arena is NULL (size
 *                  query only).
 *
 * With arena == NULL nothing touches the GPU: the call validates the trees,
 * reports the size and, when `out` is given, returns a host-only bank that
 * supports entmtp_bank_info / entmtp_bank_export but not the kernels (they
 * return ENTMTP_EINVAL for it).  With an arena, the host image is uploaded
 * with one copy on `stream`, which this call then synchronises (the bank is
 * built once, off the hot path).  Per tree the arena holds:
 *   parent int32[T], depth int32[T] (position offset of each node),
 *   mask uint32[T][ENTMTP_MASK_WORDS] (bit j of row i, word j/32 bit j%32,
 *   set iff node j is node i or an ancestor of it; bits >= T are zero),
 *   path int32[T][D+1] (ancestor of node i at depth k, -1 past depth(i)),
 *   retrieve int32[n_leaves][D+1] (path rows of the leaves, ascending),
 * where D is the tree's depth.  The bank is immutable after the build; the
 * caller keeps the arena alive while the bank is used.
 * Errors: EINVAL (null pointers, n_trees < 1), ETREE, ERANGE, ENOSPC, EHIP.
 */
int32_t entmtp_bank_build(const int32_t* parents_host, const int32_t* sizes_host,
                          int32_t n_trees, void* arena, size_t arena_bytes,
                          size_t* arena_needed, void* stream, entmtp_bank** out);

/* Free the host handle (not the caller's arena).  NULL is accepted. */
int32_t entmtp_bank_destroy(entmtp_bank* bank);

/* Number of trees in the bank (or a negative status). */
int32_t entmtp_bank_size(const entmtp_bank* bank);

/* Host outs (each optional): node count, depth and leaf count of tree `topo`. */
int32_t entmtp_bank_info(const entmtp_bank* bank, int32_t topo, int32_t* T,
                         int32_t* D, int32_t* n_leaves);

/* Copy tree `topo`'s buffers to host memory (each pointer optional), with the
 * shapes documented at entmtp_bank_build: mask [T][ENTMTP_MASK_WORDS], depth
 * [T], path [T][D+1], retrieve [n_leaves][D+1], parent [T]. */
int32_t entmtp_bank_export(const entmtp_bank* bank, int32_t topo, uint32_t* mask,
                           int32_t* depth, int32_t* path, int32_t* retrieve,
                           int32_t* parent);

/* ------------------------------------------------------------------------ */
/* Tree-masked attention (§2.3 single sparse verification pass; §3.2: the     */
/* mask size is part of the per-step verifier cost).                          */
/* ------------------------------------------------------------------------ */

/* Workspace bytes entmtp_tree_attn needs for these sizes (0 on bad sizes).
 * Non-decreasing in T and prefix_len, so one query at the largest tree and
 * the cache capacity covers every later call. */
size_t entmtp_tree_attn_workspace(int32_t T, int32_t Hq, int32_t Hkv, int32_t d,
                                  int32_t prefix_len);

/*
 * One attention layer over the draft tree `topo` of `bank`.
 *
 *   q        [T][Hq][d] bf16: queries of the tree nodes.
 *   k_tree   [T][Hkv][d] bf16, v_tree [T][Hkv][d] bf16: the nodes' keys/values.
 *   k_cache, v_cache  [Hkv][cap][d] bf16: one layer's cache; slots
 *            [0, prefix_len) hold the prefix (keys already rotated).
 *   out      [T][Hq][d] bf16.
 *   workspace  device scratch of at least entmtp_tree_attn_workspace() bytes;
 *            it holds the split partials of one call, so calls that share a
 *            workspace must be ordered, never concurrent.
 *
 * The call writes the tree's keys and values into cache slots
 * [prefix_len, prefix_len + T) and computes, for node i and query head h
 * (KV head g = h / (Hq / Hkv)), softmax-weighted values over the keys at
 * slots [0, prefix_len) and prefix_len + j for every node j on i's
 * root-to-node path, with logits scale * (q . k) and fp32 softmax.  When
 * rope_theta > 0, q_i and k_i are first rotated to position
 * prefix_len + depth(i) (pairs (c, c + d/2) turned by the angle
 * pos * rope_theta^(-2c/d), computed in fp64; the rotated key is rounded to
 * bf16 once, nearest-even); rope_theta == 0 disables the rotation.
 * Requirements: d == ENTMTP_HEAD_DIM, Hq % Hkv == 0 (else ERANGE),
 * cap >= prefix_len + T (else ERANGE), prefix_len >= 0.
 * Errors: EINVAL, ERANGE, ENOSPC (workspace), EHIP.
 */
int32_t entmtp_tree_attn(const entmtp_bank* bank, int32_t topo, const entmtp_bf16* q,
                         const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                         entmtp_bf16* k_cache, entmtp_bf16* v_cache, int32_t cap,
                         int32_t prefix_len, int32_t Hq, int32_t Hkv, int32_t d,
                         float scale, float rope_theta, entmtp_bf16* out,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * Allocation-free form of entmtp_tree_attn, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops or harnesses
 * that forbid allocation).  Same arguments, computation and outputs as
 * entmtp_tree_attn, without the workspace: the call uses a static device
 * array of ENTMTP_NOALLOC_SCRATCH_BYTES that the library holds on every
 * device it runs on until the process ends (its device address is looked up
 * once per device, on the first call made with that device current).
 * It accepts exactly the calls with
 *   entmtp_tree_attn_workspace(T, Hq, Hkv, d, prefix_len) <= ENTMTP_NOALLOC_SCRATCH_BYTES
 * and rejects any other with ENOSPC before launching anything.  It allocates
 * and frees nothing.  The array keeps the last call's contents; nothing in it
 * has to start at zero (every call writes what it reads).  All calls on one
 * device share the array: calls that can overlap on one device (on streams
 * not ordered with each other, or from several host threads) race, and the
 * caller must order them.
 * Errors: EINVAL, ERANGE, ENOSPC (sizes beyond the array), EHIP.
 */
#define ENTMTP_NOALLOC_SCRATCH_BYTES (96u * 1024u * 1024u)
int32_t entmtp_tree_attn_noalloc(const entmtp_bank* bank, int32_t topo, const entmtp_bf16* q,
                                 const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                                 entmtp_bf16* k_cache, entmtp_bf16* v_cache, int32_t cap,
                                 int32_t prefix_len, int32_t Hq, int32_t Hkv, int32_t d,
                                 float scale, float rope_theta, entmtp_bf16* out, void* stream);

/*
 * Batched form: B sequences (1 <= B <= ENTMTP_B_MAX), each with its own tree
 * (topo[b]), prefix length (prefix_len[b]) and cache (k_caches[b],
 * v_caches[b], each [Hkv][cap][d] bf16) -- the per-sequence tree choice of §4
 * applied to every sequence of a batch.  topo, prefix_len, k_caches and
 * v_caches are HOST arrays of B entries (the caches they list are device
 * buffers); the scheduler runs on the host, so the grid follows the trees.
 * q, k_tree, v_tree and out hold the sequences' tree rows back to back: the
 * rows of sequence b start at row_off[b] = T(topo[0]) + ... + T(topo[b-1])
 * (q / out rows are [Hq][d], k_tree / v_tree rows [Hkv][d]).  Each sequence
 * is computed exactly as entmtp_tree_attn computes it.
 *   workspace  device scratch of at least
 *              entmtp_tree_attn_batched_workspace(B, T_max, Hq, Hkv, d,
 *              max_prefix_len) bytes, where T_max and max_prefix_len bound
 *              every sequence's tree size and prefix length.
 * Errors: EINVAL, ERANGE, ENOSPC, EHIP (the failing sequence is named).
 */
size_t entmtp_tree_attn_batched_workspace(int32_t B, int32_t T_max, int32_t Hq, int32_t Hkv,
                                          int32_t d, int32_t max_prefix_len);
int32_t entmtp_tree_attn_batched(const entmtp_bank* bank, int32_t B, const int32_t* topo,
                                 const int32_t* prefix_len, const entmtp_bf16* q,
                                 const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                                 entmtp_bf16* const* k_caches, entmtp_bf16* const* v_caches,
                                 int32_t cap, int32_t Hq, int32_t Hkv, int32_t d, float scale,
                                 float rope_theta, entmtp_bf16* out, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * Batched form with the per-sequence choices in DEVICE memory (the
 * per-sequence tree choice of §4 made on the GPU, or by a caller that keeps
 * its schedule there): topo[B], prefix_len[B] and row_off[B + 1] are device
 * int32 arrays read by the kernels, so the call never waits for them;
 * sequence b's tree rows are rows row_off[b] .. row_off[b] + T - 1 of q /
 * k_tree / v_tree / out (T = its tree's size; they must lie in
 * [row_off[b], row_off[b + 1]), so sequences may leave gaps), which hold
 * rows_cap rows.  k_caches / v_caches are HOST
 * arrays of B device pointers, each [Hkv][cap][d] bf16.  Each sequence is
 * computed exactly as entmtp_tree_attn_batched computes it for the same
 * trees and prefix lengths (the kernels derive the same plan).  The grids
 * are sized on the host for the bank's largest plan (trees up to the
 * bank's largest, prefix lengths up to cap - T).  A sequence whose topo[b]
 * lies outside the bank, whose prefix_len[b] is negative or leaves fewer
 * than T free cache slots, or whose tree rows do not lie in [row_off[b],
 * row_off[b + 1]) and rows_cap computes nothing (its out rows and cache are
 * left as they were); the host cannot see device values, so that is not an
 * error.
 *   workspace  device scratch of at least
 *              entmtp_tree_attn_batched_device_workspace(bank, B, Hq, Hkv, d,
 *              cap) bytes (0 for invalid arguments).
 * Requirements: the bank names at most 32 trees; otherwise as
 * entmtp_tree_attn_batched.
 * Errors (host-checked): EINVAL, ERANGE, ENOSPC, EHIP.
 */
size_t entmtp_tree_attn_batched_device_workspace(const entmtp_bank* bank, int32_t B, int32_t Hq,
                                                 int32_t Hkv, int32_t d, int32_t cap);
int32_t entmtp_tree_attn_batched_device(const entmtp_bank* bank, int32_t B, const int32_t* topo,
                                        const int32_t* prefix_len, const int32_t* row_off,
                                        int32_t rows_cap, const entmtp_bf16* q,
                                        const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                                        entmtp_bf16* const* k_caches,
                                        entmtp_bf16* const* v_caches, int32_t cap, int32_t Hq,
                                        int32_t Hkv, int32_t d, float scale, float rope_theta,
                                        entmtp_bf16* out, void* workspace,
                                        size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* LM-head verification logits (§2.2: next-token distribution softmax(W h);  */
/* §2.3: one verification pass for all tree nodes).                           */
/* ------------------------------------------------------------------------ */

/*
 * logits[i][v] = sum_k hidden[i][k] * w_lm[v][k]   (fp32 accumulation)
 *
 *   hidden  [T][hid] bf16: final hidden states of the tree nodes.
 *   w_lm    [V][hid] bf16: LM-head weight (nn.Linear layout).
 *   logits  [T][V] fp32.
 * Requirements: 1 <= T <= 4096, hid % 8 == 0, V >= 1, pointers 16-byte aligned.
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_verify_logits(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                             int32_t T, int32_t hid, int32_t V, float* logits,
                             void* stream);

/*
 * Fused form of entmtp_verify_logits followed by entmtp_logit_stats: the
 * LM-head kernel also reduces every workgroup's vocabulary slice to per-node
 * softmax partials (largest raw logit with its lowest index, and the sums
 * sum e^(y-m), sum (y-m) e^(y-m) for y = inv_temp * z), which a small kernel
 * then combines per node, so the logits are not read back.  Outputs and their
 * meaning are those of the two separate calls (entropy / top1p / argmax may
 * each be NULL; logits [T][V] fp32 is written unless it is NULL, which is
 * allowed when hid is a multiple of 512 -- the statistics then come from the
 * accumulators alone and no logits reach memory).
 *   workspace   device scratch of at least
 *               entmtp_verify_logits_stats_workspace(T, hid, V) bytes, 16-byte
 *               aligned (partials, overwritten by every call).
 * Errors: EINVAL, ENOSPC (workspace), EHIP.
 */
size_t entmtp_verify_logits_stats_workspace(int32_t T, int32_t hid, int32_t V);
int32_t entmtp_verify_logits_stats(const entmtp_bf16* hidden, const entmtp_bf16* w_lm, int32_t T,
                                   int32_t hid, int32_t V, float inv_temp, float* logits,
                                   float* entropy, float* top1p, int32_t* argmax,
                                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * The two halves of entmtp_verify_logits_stats, for callers that time or
 * schedule them separately.  Available when hid is a multiple of 512 (the
 * streaming LM-head kernel); entmtp_stats_partials_bytes returns 0 otherwise
 * and entmtp_verify_logits_partials then fails with EINVAL.
 *   partials   device buffer of entmtp_stats_partials_bytes(T, hid, V) bytes,
 *              16-byte aligned; written by the first call, read by the second
 *              (same device, same V).
 *   logits     may be NULL (statistics only).
 */
size_t entmtp_stats_partials_bytes(int32_t T, int32_t hid, int32_t V);
int32_t entmtp_verify_logits_partials(const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                                      int32_t T, int32_t hid, int32_t V, float inv_temp,
                                      float* logits, void* partials, size_t partials_bytes,
                                      void* stream);
int32_t entmtp_stats_finalize(const void* partials, int32_t T, int32_t V, float inv_temp,
                              float* entropy, float* top1p, int32_t* argmax, void* stream);

/* ------------------------------------------------------------------------ */
/* Per-node softmax statistics (§4: the scheduler reads the top-1            */
/* probability p0 at the verifier's last position; §3 / App. A: entropy).    */
/* ------------------------------------------------------------------------ */

/*
 * For each row i of logits [T][V] (fp32), with y = inv_temp * z:
 *   argmax[i]  lowest index attaining max(z)              (int32)
 *   top1p[i]   exp(max y) / sum_v exp(y_v) = 1 / Z         (fp32)
 *   entropy[i] -sum_v p_v ln p_v = ln Z - sum (y_v - m) e^(y_v - m) / Z, nats
 * Each output pointer may be NULL to skip it.  inv_temp must be > 0.
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_logit_stats(const float* logits, int32_t T, int32_t V, float inv_temp,
                           float* entropy, float* top1p, int32_t* argmax, void* stream);

/* ------------------------------------------------------------------------ */
/* Acceptance (§2.1 left-to-right acceptance, greedy case; §5.1 accept       */
/* length).                                                                   */
/* ------------------------------------------------------------------------ */

/*
 * Greedy verification of tree `topo`: node i >= 1 is accepted when
 * draft_tokens[i] == argmax[parent(i)] and its parent is accepted (the root
 * always is).  best = the deepest accepted node, lowest index among equals.
 *
 *   draft_tokens  int32[T] (entry 0, the root's, is ignored)
 *   argmax        int32[T] target greedy tokens (from entmtp_logit_stats)
 *   top1p         fp32[T] or NULL
 *   accept_len    int32 out: depth(best) = accepted draft tokens
 *   path          int32[D+1] out: root-to-best chain, -1 after accept_len
 *   bonus         int32 out: argmax[best]
 *   best_top1p    fp32 out or NULL: top1p[best] (the scheduler's feature)
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_accept(const entmtp_bank* bank, int32_t topo, const int32_t* draft_tokens,
                      const int32_t* argmax, const float* top1p, int32_t* accept_len,
                      int32_t* path, int32_t* bonus, float* best_top1p, void* stream);

/*
 * Typical acceptance (the verification condition the paper keeps from Hydra:
 * temperature, posterior threshold eps, mixing coefficient alpha, §5.1-§5.2;
 * the rule is the published typical acceptance of Medusa/Hydra).  Node i >= 1
 * is locally acceptable when its draft token's probability under its parent's
 * distribution p = softmax(z[parent] * inv_temp) exceeds
 * min(eps, alpha * exp(-H(p))), and accepted when every ancestor is too.
 * The answer is the deepest accepted node; among several of that depth, the
 * one whose path's draft tokens are jointly most likely (largest sum of
 * log p(draft) from the root, decided in fp32; then the lowest index), the
 * published rule's choice among equally long candidates.  Outputs (accept
 * length, path with -1 past it, bonus = argmax at the chosen node,
 * best_top1p) are as for entmtp_accept; path has D + 1 entries.
 *
 * entmtp_draft_logits computes what the test needs beyond the statistics:
 * z_draft[i] = X[parent(i)] . W[draft_tokens[i]] and z_top[i] = X[parent(i)] .
 * W[argmax[parent(i)]] (fp32, device [T]; 0 for the root; -inf for a draft
 * token outside [0, V)).  hidden [T][hid] and w_lm [V][hid] bf16, 16-byte
 * aligned, hid % 8 == 0.
 *
 * entmtp_accept_typical takes those and the statistics entmtp_logit_stats /
 * entmtp_verify_logits_stats produced with the same inv_temp (entropy in
 * nats, top1p, argmax): p(draft) = exp((z_draft - z_top) * inv_temp) *
 * top1p[parent].  eps, alpha >= 0.
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_draft_logits(const entmtp_bank* bank, int32_t topo, const entmtp_bf16* hidden,
                            const entmtp_bf16* w_lm, int32_t hid, int32_t V,
                            const int32_t* draft_tokens, const int32_t* argmax, float* z_draft,
                            float* z_top, void* stream);
int32_t entmtp_accept_typical(const entmtp_bank* bank, int32_t topo, const int32_t* draft_tokens,
                              const int32_t* argmax, const float* z_draft, const float* z_top,
                              const float* entropy, const float* top1p, float inv_temp, float eps,
                              float alpha, int32_t* accept_len, int32_t* path, int32_t* bonus,
                              float* best_top1p, void* stream);

/*
 * Batched form: workgroup b accepts tree topo[b] (HOST array of B entries,
 * 1 <= B <= ENTMTP_B_MAX) of sequence b.  draft_tokens, argmax and top1p hold
 * the sequences' rows back to back (rows of sequence b start at
 * T(topo[0]) + ... + T(topo[b-1]), the layout entmtp_tree_attn_batched uses;
 * the LM head and statistics run over those rows unchanged).  Outputs, one
 * per sequence: accept_len[B], bonus[B], best_top1p[B] (may be NULL), and
 * path [B][path_capacity] (node indices local to the sequence's tree, -1 past
 * its accept length); path_capacity >= 1 + every tree's depth.
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_accept_batched(const entmtp_bank* bank, int32_t B, const int32_t* topo,
                              const int32_t* draft_tokens, const int32_t* argmax,
                              const float* top1p, int32_t* accept_len, int32_t* path,
                              int32_t path_capacity, int32_t* bonus, float* best_top1p,
                              void* stream);

/*
 * Batched form with the trees and rows in DEVICE memory: topo[B] and
 * row_off[B + 1] are device int32 arrays; sequence b's rows of draft_tokens,
 * argmax and top1p are row_off[b] .. row_off[b] + T - 1 (within
 * [row_off[b], row_off[b + 1]) and the rows_cap rows they hold).  Outputs as
 * entmtp_accept_batched (equal for the same trees and rows).  A sequence
 * whose topo[b] lies outside the bank, whose tree rows do not lie in
 * [row_off[b], row_off[b + 1]) and rows_cap, or whose tree's depth + 1
 * exceeds path_capacity is not verified: accept_len[b] = -1, bonus[b] = -1,
 * its path row -1 and best_top1p[b] = 0 (entmtp_kv_compact_batched_device
 * then moves nothing for it).
 * Requirements: the bank names at most 32 trees, 1 <= path_capacity <= 256.
 * Errors (host-checked): EINVAL, ERANGE, EHIP.
 */
int32_t entmtp_accept_batched_device(const entmtp_bank* bank, int32_t B, const int32_t* topo,
                                     const int32_t* row_off, int32_t rows_cap,
                                     const int32_t* draft_tokens, const int32_t* argmax,
                                     const float* top1p, int32_t* accept_len, int32_t* path,
                                     int32_t path_capacity, int32_t* bonus, float* best_top1p,
                                     void* stream);

/* ------------------------------------------------------------------------ */
/* KV-cache update of the accepted path (§3.2 decode loop).                   */
/* ------------------------------------------------------------------------ */

/*
 * For every layer l < n_layers and KV head g < Hkv, and j = 0..a with
 * a = *accept_len (read on the device):
 *   cache[l][g][prefix_len + j] <- cache[l][g][prefix_len + path[j]]
 * for both k_cache and v_cache, all reads before any write (a source slot may
 * be another row's destination).  Layer l's cache starts layer_stride
 * elements after layer l-1's; each layer is [Hkv][cap][d].  Slots past
 * prefix_len + a are left as they were.  path (device int32[path_capacity])
 * and accept_len come from entmtp_accept on the same stream.  The kernel
 * clamps a to [0, min(path_capacity, ENTMTP_D_MAX + 1) - 1] and skips (leaves
 * unchanged) any row whose source or destination slot would fall outside
 * [0, cap).
 * Requirements: d % 8 == 0, 8 <= d <= 256, prefix_len >= 0, cap >= 1,
 * path_capacity >= 1, layer_stride >= Hkv * cap * d when n_layers > 1,
 * 16-byte aligned caches.
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_kv_compact(const int32_t* path, int32_t path_capacity,
                          const int32_t* accept_len, int32_t prefix_len,
                          entmtp_bf16* k_cache, entmtp_bf16* v_cache, int32_t n_layers,
                          int64_t layer_stride, int32_t Hkv, int32_t cap, int32_t d,
                          void* stream);

/*
 * Batched form: sequence b (1 <= B <= ENTMTP_B_MAX) keeps the path in row b
 * of path [B][path_capacity] (device) with accept length accept_len[b]
 * (device), in its own cache k_caches[b] / v_caches[b] (HOST array of device
 * pointers) at prefix length prefix_len[b] (HOST array); every sequence is
 * compacted exactly as entmtp_kv_compact compacts one, in all n_layers
 * layers.  Errors: EINVAL, EHIP.
 */
int32_t entmtp_kv_compact_batched(int32_t B, const int32_t* path, int32_t path_capacity,
                                  const int32_t* accept_len, const int32_t* prefix_len,
                                  entmtp_bf16* const* k_caches, entmtp_bf16* const* v_caches,
                                  int32_t n_layers, int64_t layer_stride, int32_t Hkv,
                                  int32_t cap, int32_t d, void* stream);

/*
 * Batched form with the prefix lengths in DEVICE memory: prefix_len[B] is a
 * device int32 array (k_caches / v_caches stay HOST arrays of device
 * pointers); otherwise as entmtp_kv_compact_batched.  A sequence whose
 * prefix_len[b] lies outside [0, cap) is left unchanged.
 * Errors (host-checked): EINVAL, EHIP.
 */
int32_t entmtp_kv_compact_batched_device(int32_t B, const int32_t* path, int32_t path_capacity,
                                         const int32_t* accept_len, const int32_t* prefix_len,
                                         entmtp_bf16* const* k_caches,
                                         entmtp_bf16* const* v_caches, int32_t n_layers,
                                         int64_t layer_stride, int32_t Hkv, int32_t cap,
                                         int32_t d, void* stream);

/* ------------------------------------------------------------------------ */
/* Scheduler policy (§4 "Policy"), host only.                                 */
/* ------------------------------------------------------------------------ */

/* Hysteretic ladder over a bank sorted by size: climb one rung when
 * s > tau_on, descend one when s <= tau_off, else stay; clamped to
 * [0, n_rungs).  Returns the next rung (or a negative status). */
int32_t entmtp_ladder_next(int32_t rung, int32_t n_rungs, float s, float tau_on,
                           float tau_off);

/* The same ladder for a batch of sequences, each with its own rung (§4
 * "Policy", applied per sequence): rung[B] (host, in/out) moves one step on
 * s[B] (host), the per-sequence top-1 probability the acceptance reports.
 * Every rung is checked before any is changed; on an error rung[] is left as
 * it was.  Errors: EINVAL (B < 0, null array, n_rungs < 1, tau_off > tau_on,
 * a rung outside [0, n_rungs)). */
int32_t entmtp_ladder_next_batched(int32_t B, int32_t* rung, const float* s, int32_t n_rungs,
                                   float tau_on, float tau_off);

/*
 * Speculative-sampling verification (§2.1: keep a draft token t with
 * probability min(1, p(t) / p_hat(t)), else draw a replacement from
 * norm(max(0, p - p_hat)) and drop the rest).  On a tree: from the root, with
 * r = p at the current node, the node's children are tried in index (rank)
 * order, all drafted from the node's draft distribution q[node]; child c
 * passes when u_accept[c] * q(t_c) < r(t_c) (with q(t_c) = 0: when
 * r(t_c) > 0) and becomes the current node (r = p at it); a child that fails
 * replaces r by norm(max(0, r - q[node])) (kept as is if that has no mass)
 * before the next sibling.  With no child passing, or at a leaf, the bonus
 * token is drawn from r with u_sample[node]: the smallest index b whose
 * cumulative mass (vocabulary in index order) exceeds u_sample * total.  A
 * chain tree gives exactly the §2.1 rule.  A draft token outside [0, V)
 * never passes (the residual update follows as for any rejection).
 *   logits   device fp32 [T][V]: the target's logits per node, p =
 *            softmax(logits * inv_temp)
 *   argmax, top1p  device [T]: the statistics of those logits at the same
 *            inv_temp (entmtp_logit_stats / entmtp_verify_logits_stats), so
 *            that p(v) = exp((z_v - z_argmax) * inv_temp) * top1p needs no
 *            pass over the vocabulary
 *   q        device fp32 [T][V]: the draft distribution node i's children
 *            were drawn from (rows sum to 1)
 *   u_accept, u_sample  device fp32 [T]: uniforms in [0, 1) (the method's
 *            random numbers, supplied by the caller)
 *   workspace  device fp32 [V] scratch (the residual), used by this call only
 *   accept_len, path [D+1] (entries past accept_len -1), bonus: as for
 *            entmtp_accept
 * Errors: EINVAL, EHIP.
 */
int32_t entmtp_accept_stochastic(const entmtp_bank* bank, int32_t topo,
                                 const int32_t* draft_tokens, const float* logits, const float* q,
                                 int32_t V, float inv_temp, const int32_t* argmax,
                                 const float* top1p, const float* u_accept,
                                 const float* u_sample, float* workspace, int32_t* accept_len,
                                 int32_t* path, int32_t* bonus, void* stream);

/* ------------------------------------------------------------------------ */
/* Acceptance frontier (§3.1, Algorithm 1: the scoring step of the greedy     */
/* offline tree search)                                                       */
/* ------------------------------------------------------------------------ */

/*
 * NextChildren(T, D) of Algorithm 1 (§3.1; the paper does not spell it out):
 * every node of T whose depth is below max_depth, the root included, proposes
 * its next-ranked child (rank = its current number of children, the greedy
 * tree-growing step of Medusa/Hydra tree lists).  Builds the joint tree
 * T u F that entmtp_frontier_score scores: T's nodes keep their indices, the
 * candidates follow in node order of their parents.  Host only.
 *   parent       HOST int32[T], parent[0] = -1, 0 <= parent[i] < i
 *   T            1 <= T
 *   max_depth    D >= 0 (a candidate's depth is at most D)
 *   joint_parent HOST int32[joint_capacity] out: the parent array of T u F
 *   in_tree      HOST uint8[joint_capacity] out (may be NULL): 1 for T's nodes,
 *                0 for the candidates
 *   joint_T      HOST int32 out: T + |F|
 * Errors: EINVAL (NULL pointer, bad parent array, max_depth < 0), ENOSPC
 * (T + |F| > joint_capacity; *joint_T still receives T + |F| and nothing
 * else is written).
 */
int32_t entmtp_frontier_tree(const int32_t* parent, int32_t T, int32_t max_depth,
                             int32_t* joint_parent, uint8_t* in_tree, int32_t joint_capacity,
                             int32_t* joint_T);

/*
 * Scores every one-node augmentation T u {nu} of a draft tree T from one
 * rollout of the joint tree T u F, and picks the node Algorithm 1 adds.
 *   bank, topo   the joint tree (a bank tree); nodes are ranked among their
 *                parent's children in index order, and a node's rank sum is
 *                the sum of the ranks on its root-to-node path (the Medusa
 *                tuple of the node, added up)
 *   in_tree      device uint8[T]: nonzero for the nodes of T (the root counts
 *                as one whatever its flag), 0 for the candidates
 *   n_samples    S >= 1 verifications of the joint tree (S x depth < 2^31)
 *   local_ok     device uint8[S][T] or NULL: nonzero when node i's draft token
 *                passes the local test in sample s (any acceptance rule); when
 *                NULL, draft_tokens and argmax (device int32[S][T]) decide it
 *                greedily: draft_tokens[s][i] == argmax[s][parent(i)]
 *   sums         device int32[T] out: for a candidate, the accept length of
 *                T u {nu} summed over the samples -- per sample the larger of
 *                T's accept length (its deepest accepted node) and depth(nu)
 *                when nu and its ancestors are accepted; for a node of T,
 *                T's own accept length summed
 *   best         device int32[1] out: the candidate with the largest sum, then
 *                the smaller rank sum, then the smaller depth, then the lower
 *                index; -1 without candidates
 * Errors: EINVAL, ERANGE, EHIP.
 */
int32_t entmtp_frontier_score(const entmtp_bank* bank, int32_t topo, const uint8_t* in_tree,
                              int32_t n_samples, const uint8_t* local_ok,
                              const int32_t* draft_tokens, const int32_t* argmax, int32_t* sums,
                              int32_t* best, void* stream);

/* ------------------------------------------------------------------------ */
/* One verification step, end to end (§4, the decode loop with the tree      */
/* scheduler and its "Cost" paragraph: verify the chosen tree, accept, update */
/* the cache, read one scalar back to pick the next tree).                    */
/* ------------------------------------------------------------------------ */

/*
 * Fixed part of a decode loop, validated once by entmtp_step_create.  All
 * pointers are device pointers owned by the caller and must stay valid while
 * the step object is used.
 *   n_layers, Hq, Hkv, d, scale, rope_theta   as for entmtp_tree_attn; layer l
 *              of the cache starts at k_cache + l * cache_layer_stride (same for
 *              v_cache), each layer [Hkv][cap][d] bf16
 *   tree_rows  rows reserved per layer for the per-step tree inputs: q of
 *              layer l starts at q + l * tree_rows * Hq * d, k_tree / v_tree at
 *              + l * tree_rows * Hkv * d, out at + l * tree_rows * Hq * d;
 *              at least the largest T in the bank
 *   w_lm, hid, V, inv_temp   the LM head and the statistics temperature as for
 *              entmtp_verify_logits_stats (hid a multiple of 512)
 *   logits [tree_rows][V] fp32, or NULL to keep no logits (the statistics
 *              and acceptance do not need them); entropy, top1p [tree_rows]
 *              fp32; argmax [tree_rows] int32   outputs of the LM head and
 *              statistics
 *   accept_len [1], bonus [1] int32, best_top1p [1] fp32, path [path_capacity]
 *              int32 (1 + the largest depth in the bank <= path_capacity <=
 *              ENTMTP_D_MAX + 1)   outputs of acceptance, as for entmtp_accept;
 *              every step writes all path_capacity entries (-1 past its
 *              accept length, whatever the depth of its tree)
 *   workspace  scratch of entmtp_step_workspace() bytes, 256-byte aligned,
 *              used by this step object only (it holds attention partials,
 *              statistics partials and the device-scheduled state, which
 *              entmtp_step_create initialises on the stream)
 *   stream     the HIP stream every launch goes to (NULL: the null stream)
 *   tau_on, tau_off   thresholds of the hysteretic ladder (§4 "Policy") for
 *              device-scheduled steps, tau_off <= tau_on (unused otherwise)
 *   device_prefix_fixed   0: device-scheduled steps advance the prefix by the
 *              accepted tokens (the decode loop); 1: every device-scheduled
 *              step verifies at the prefix length entmtp_step_device_start
 *              set (a fixed position, for measuring one shape)
 */
typedef struct entmtp_step_config {
  int32_t n_layers, Hq, Hkv, d, cap, tree_rows;
  float scale, rope_theta;
  entmtp_bf16* k_cache;
  entmtp_bf16* v_cache;
  int64_t cache_layer_stride;
  const entmtp_bf16* w_lm;
  int32_t hid, V;
  float inv_temp;
  float* logits;
  float* entropy;
  float* top1p;
  int32_t* argmax;
  int32_t* accept_len;
  int32_t* bonus;
  float* best_top1p;
  int32_t* path;
  int32_t path_capacity;
  void* workspace;
  size_t workspace_bytes;
  void* stream;
  float tau_on, tau_off;
  int32_t device_prefix_fixed;
} entmtp_step_config;

typedef struct entmtp_step entmtp_step;

/* Workspace bytes for entmtp_step_create with this bank and configuration
 * (attention partials for the largest prefix that fits the cache, plus the
 * LM-head statistics partials); 0 when the configuration is invalid. */
size_t entmtp_step_workspace(const entmtp_bank* bank, const entmtp_step_config* cfg);

/* Validates cfg against the (device) bank, copies it, and allocates the small
 * pinned host record that acceptance publishes its result to.  The library
 * owns *out; release it with entmtp_step_destroy after the stream is idle.
 * Errors: EINVAL, ERANGE, ENOSPC, EHIP. */
int32_t entmtp_step_create(const entmtp_bank* bank, const entmtp_step_config* cfg,
                           entmtp_step** out);
void entmtp_step_destroy(entmtp_step* step);

/*
 * Enqueues one verification step for tree `topo` at prefix length prefix_len,
 * asynchronously, as two chains:
 *   on the configured stream   the LM head with fused statistics partials,
 *              then the statistics merge and greedy acceptance (one launch
 *              for trees of up to 32 nodes, two for larger ones); acceptance
 *              also publishes its result (accept_len, bonus, best_top1p and
 *              the accepted path) to pinned host memory
 *   on a side stream the step object owns, ordered after everything enqueued
 *   on the configured stream before this call
 *              the compaction of the previous step (the one whose result
 *              entmtp_step_wait read last, at that step's prefix length), then
 *              for each layer entmtp_tree_attn (writes K/V slots [L, L+T))
 * Nothing on the configured stream waits for the side stream: the LM head of
 * the next step runs beside this step's compaction and attention.  The
 * compaction of a step is therefore enqueued by the next launch, or by
 * entmtp_step_flush, and the cache and `out` are complete on the configured
 * stream only after entmtp_step_flush.
 * Every launch must be followed by entmtp_step_wait before the next launch
 * (the compaction takes the accepted path from the host record).
 * Per-step inputs (device): q, k_tree, v_tree, out laid out with tree_rows
 * rows per layer; hidden [T][hid] bf16; draft_tokens [T] int32; w_lm the
 * LM-head weight for this step ([V][hid] bf16, 16-byte aligned; NULL: the
 * configured one).
 * ev_lm_begin / ev_lm_end: optional hipEvent_t recorded on the stream right
 * before and after the LM-head launch (NULL: none).  With events, a one-lane
 * gate kernel goes ahead of ev_lm_begin and holds the stream (at most 2 ms)
 * until the host has enqueued the LM head and ev_lm_end, so the pair brackets
 * the kernel rather than the host's launch call on an idle stream.
 * Requirements: prefix_len >= 0, prefix_len + T <= cap.
 * Errors: EINVAL (also: the previous result was not read), ERANGE, EHIP (a
 * failed launch leaves the step unusable for entmtp_step_wait until the next
 * successful launch).
 */
int32_t entmtp_step_launch(entmtp_step* step, int32_t topo, int32_t prefix_len,
                           const entmtp_bf16* q, const entmtp_bf16* k_tree,
                           const entmtp_bf16* v_tree, entmtp_bf16* out,
                           const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                           const int32_t* draft_tokens, void* ev_lm_begin, void* ev_lm_end);

/*
 * Enqueues the LM head of the next host-scheduled step ahead of its launch,
 * so that the launch, issued once the host has read the previous result and
 * chosen the tree (§4 "Policy"), only has to release work already in the
 * queue.  On the configured stream, after everything enqueued so far: the
 * fork point of the next step's cache chain, a one-lane gate kernel, and
 * the LM head with fused statistics partials for rows [0, T_bound) of
 * `hidden`.  The gate holds the stream until entmtp_step_wait has read the
 * pending step's result (or the next entmtp_step_launch or entmtp_step_flush
 * comes first), or for at most 2 ms; the LM head's inputs are fixed here, so
 * a gate that times out only lets it start early.
 * The next entmtp_step_launch then uses this LM head when its tree has at
 * most T_bound nodes and it passes the same hidden and w_lm (it must pass
 * NULL events); otherwise it opens the gate and enqueues a fresh LM head
 * (the armed one runs unused).  With the ladder a step's tree is at most one
 * rung above the current one, so T_bound = the next larger tree's node count
 * always suffices; the extra rows cost little, since the LM head streams the
 * weights once for up to 16 / 32 / 64 / 128 rows.
 *   hidden [T_bound][hid] bf16; w_lm [V][hid] bf16 (NULL: the configured
 *   one); T_bound in [1, the bank's largest T]; ev_lm_begin / ev_lm_end:
 *   optional hipEvent_t recorded right before and after the LM head (behind
 *   the gate, so the pair brackets the kernel).
 * Ordering: the next step's cache chain starts after the work enqueued on
 * the stream before this call, and work enqueued after it queues behind the
 * armed LM head; so the next step's q, k_tree, v_tree, out and hidden must be
 * ready (or enqueued) before arming.  Only its draft tokens, which the
 * acceptance reads after the LM head, may still be enqueued in between.
 * The armed LM head writes the configured logits buffer (if any), so the
 * logits of the pending step are valid only until the gate opens or its
 * time limit ends the wait.
 * May be called while a launched step's result is pending (that is its use);
 * not while already armed or with device-scheduled steps running
 * (entmtp_step_device_start discards the arming).  Errors: EINVAL, ERANGE, EHIP.
 */
int32_t entmtp_step_arm(entmtp_step* step, const entmtp_bf16* hidden, const entmtp_bf16* w_lm,
                        int32_t T_bound, void* ev_lm_begin, void* ev_lm_end);

/*
 * Waits for the acceptance result of the latest entmtp_step_launch by polling
 * the pinned host record (no stream synchronisation: attention may still be
 * running).  Writes the accepted draft count, the bonus token and the top-1
 * probability at the accepted node (the scheduler's s, §4) to the host
 * pointers given (each may be NULL), and keeps the accepted path for the
 * step's compaction.  Gives up after timeout_s seconds with ETIMEDOUT, or
 * earlier with EHIP when the stream reports an error.
 */
int32_t entmtp_step_wait(entmtp_step* step, int32_t* accept_len, int32_t* bonus,
                         float* best_top1p, double timeout_s);

/*
 * Enqueues the compaction of the last step (for host-scheduled steps: the
 * last one whose result was read) if not yet enqueued, and joins the side
 * stream into the configured stream: work enqueued on the configured stream
 * afterwards sees every step's cache update and attention output.  Errors:
 * EINVAL (a launched host-scheduled step's result has not been read), EHIP.
 */
int32_t entmtp_step_flush(entmtp_step* step);

/*
 * Device-scheduled steps: the tree choice of §4 moved next to the statistics
 * it reads.  The acceptance kernel of a step also runs the hysteretic ladder
 * (rung + 1 when s > tau_on, rung - 1 when s <= tau_off, clamped to the bank,
 * which must be sorted by size) on s = top-1 probability at the accepted node,
 * and stores the next step's tree and prefix length (L + accept_len + 1) in
 * device memory, so the host enqueues step after step without reading
 * anything back.  The decisions are those of entmtp_ladder_next on the same s.
 *
 * entmtp_step_device_start: flushes host-scheduled steps (entmtp_step_flush)
 * and sets the device state to tree `topo` at prefix_len (asynchronously, on
 * the configured stream).  Requires a bank of trees of at most 128 nodes.
 * Errors: EINVAL, ERANGE, EHIP.
 *
 * entmtp_step_launch_device: enqueues one step for the tree the device state
 * holds (the same kernels as entmtp_step_launch, sized for the largest
 * tree), in the same two chains: the LM head and acceptance on the
 * configured stream, and on the side stream (ordered after everything the
 * caller enqueued before the call) the previous step's compaction and this
 * step's attention.  Acceptance of step t waits only for the side stream's
 * work of step t-2, so the host can enqueue steps ahead of the GPU.  As with
 * entmtp_step_launch, the last step's compaction goes out with
 * entmtp_step_flush, after which every output is complete on the configured
 * stream; accept_len and path of the configuration hold the latest step's.
 * Inputs as for entmtp_step_launch, except
 *   w_lm    the LM-head weight for this step ([V][hid] bf16, NULL: the
 *           configured one)
 *   drafts  [K][tree_rows] int32 (device): the draft tokens for every bank
 *           tree (row k for tree k; the step reads the chosen tree's row)
 *   log     device int32[log_rows][4] or NULL: row (step index since
 *           entmtp_step_device_start) % log_rows receives (tree, prefix
 *           length, accept_len, s as float bits) of the step
 * The caller sizes cap for the whole run (prefix growth included).  A step
 * whose prefix length plus tree would exceed cap computes no attention; it
 * and every later step of the run keep the tree and prefix length they had,
 * and their log rows carry accept length -1 (the host reads the overflow
 * there).
 * Errors: EINVAL (no entmtp_step_device_start yet), EHIP.
 */
int32_t entmtp_step_device_start(entmtp_step* step, int32_t topo, int32_t prefix_len);
int32_t entmtp_step_launch_device(entmtp_step* step, const entmtp_bf16* q,
                                  const entmtp_bf16* k_tree, const entmtp_bf16* v_tree,
                                  entmtp_bf16* out, const entmtp_bf16* hidden,
                                  const entmtp_bf16* w_lm, const int32_t* drafts, int32_t* log,
                                  int32_t log_rows, void* ev_lm_begin, void* ev_lm_end);

/*
 * A segment of device-scheduled steps as one HIP graph: since such steps read
 * nothing back, n_steps of them (a multiple of 16, the depth of the device
 * state ring) are captured from the configured stream (which must not be the
 * null stream) with their per-step inputs -- host arrays of n_steps device
 * pointers, w_lm may be NULL (the configured weight) -- and a final flush, so
 * that the segment depends on nothing outside it.  Each
 * entmtp_step_graph_launch then runs the segment's steps on the configured
 * stream, continuing from whatever tree and prefix length the device state
 * holds (the log rows follow the device's step count); replays of one graph
 * may follow each other, and eager steps whose number is a multiple of 16
 * (entmtp_step_graph_launch returns EINVAL otherwise: the segment's steps
 * read fixed ring slots).  *graph receives an opaque handle;
 * release it with entmtp_step_graph_destroy.  Requires
 * entmtp_step_device_start first.  Errors: EINVAL, ERANGE, EHIP.
 */
int32_t entmtp_step_device_graph(entmtp_step* step, int32_t n_steps, const entmtp_bf16* const* q,
                                 const entmtp_bf16* const* k_tree,
                                 const entmtp_bf16* const* v_tree, entmtp_bf16* const* out,
                                 const entmtp_bf16* const* hidden, const entmtp_bf16* const* w_lm,
                                 const int32_t* const* drafts, int32_t* log, int32_t log_rows,
                                 void** graph);
int32_t entmtp_step_graph_launch(entmtp_step* step, void* graph);
void entmtp_step_graph_destroy(void* graph);

#ifdef __cplusplus
}
#endif

#endif /* ENTMTP_H */
