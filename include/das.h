/*
 * das.h -- C ABI of the depth-asynchronous self-speculation (DAS) attention
 * library for AMD Instinct MI355X (gfx950).
 *
 * The library computes the policy attention of Eq. (2)-(3) of
 * "Shallow Queries, Mature Values: Depth-Asynchronous Self-Speculation for
 * Looped Transformers" over a depth-indexed, paged key/value cache, and the
 * commit of verified tokens into that cache (Sec. 3.4 and App. B.1).
 *
 *   [Pi_C, Pi_U] = softmax( Q [K_C^kappa ; K_U]^T / sqrt(d_h) + M )     Eq. (2)
 *   O            = Pi_C V_C^nu + Pi_U V_U                               Eq. (3)
 *
 * C is the verified, materialised prefix of a sequence, U the active block
 * (draft-side positions). kappa and nu are the recurrence depths at which the
 * prefix keys and values are read (Eq. (4)); block K/V always come from the
 * caller's current computation and are never read from the cache. M is the
 * causal mask: every prefix position is visible, block query i sees block
 * keys j <= i. Prefix and block positions share one softmax normaliser.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Ownership: every pointer is owned by the caller. The library allocates
 *   no device or host memory and frees nothing; its only device memory is
 *   the fixed scratch array of das_attn_policy_noalloc (one per GPU, part of
 *   the loaded code). Device pointers must stay valid until the enqueued
 *   work has completed on `stream`.
 * - Asynchrony: calls only validate arguments and enqueue kernels on
 *   `stream`; they return before the GPU work runs. Device faults surface at
 *   the caller's next synchronisation of that stream.
 * - Errors: every argument check runs on the host before any HIP call. A
 *   failed check returns a negative das_status and enqueues nothing. A
 *   failed kernel launch returns DAS_ERR_HIP; the status is that of the
 *   library's own launches, so an error left pending by the caller's earlier
 *   HIP work is neither reported as the library's nor cleared. Requests whose
 *   launch grid would exceed what HIP accepts (2^32 - 1 work-items along a
 *   grid dimension) are rejected with DAS_ERR_SHAPE. No exception and no
 *   exit() crosses this boundary.
 * - Device-side range checks: when `dev_error` in das_batch is non-NULL the
 *   kernels OR bits into it (DAS_DEVERR_*) for out-of-range page ids,
 *   prefix lengths or commit counts, and skip the offending data instead of
 *   reading or writing out of bounds.
 * - Reentrancy: apart from the per-device scratch address of
 *   das_attn_policy_noalloc (set once, under a lock) the library keeps no
 *   global state; calls from several host threads are safe. Concurrent calls that share a workspace or write the
 *   same cache rows race on the device, as any two kernels writing the same
 *   memory would.
 * - Alignment: the kernels move K/V/Q/O rows with 16-byte accesses, so
 *   k_pool, v_pool, q, k_blk, v_blk, out, k_new and v_new must be 16-byte
 *   aligned (any allocation, or a view starting on a row, is); int32 and
 *   fp32 arrays must be 4-byte aligned. Otherwise DAS_ERR_ALIGN.
 * - Numerics: scale is 1/sqrt(head_dim). Query head h reads KV head
 *   h / (Hq / Hkv). Accumulation is fp32; outputs are rounded to the input
 *   dtype (round to nearest even).
 */
#ifndef DAS_H
#define DAS_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Largest supported recurrence depth R; depths are 1-based (1..R). */
#define DAS_MAX_DEPTH 64
/* Tokens per cache page. */
#define DAS_PAGE_TOKENS 64
/* Largest block (draft or verifier input) width w. */
#define DAS_MAX_BLOCK 64

typedef enum das_status {
  DAS_OK = 0,
  DAS_ERR_NULL = -1,        /* a required pointer is NULL                     */
  DAS_ERR_SHAPE = -2,       /* a size is out of range or inconsistent         */
  DAS_ERR_DEPTH = -3,       /* depth outside 1..R or not stored in the cache  */
  DAS_ERR_DTYPE = -4,       /* unknown element type                           */
  DAS_ERR_WORKSPACE = -5,   /* workspace missing or smaller than required     */
  DAS_ERR_HIP = -6,         /* a HIP launch failed                            */
  DAS_ERR_UNSUPPORTED = -7, /* valid request that this build does not handle  */
  DAS_ERR_ALIGN = -8        /* a device array is not aligned as required      */
} das_status;

typedef enum das_dtype { DAS_F32 = 0, DAS_BF16 = 1 } das_dtype;

/* Bits OR-ed into das_batch.dev_error by the kernels. */
#define DAS_DEVERR_PAGE 1u       /* block_table entry outside [0, num_pages)      */
#define DAS_DEVERR_PREFIX 2u     /* prefix_len[b] < 0 or beyond the table's pages */
#define DAS_DEVERR_COMMIT 4u     /* num_new[b] outside [0, w_max], or the commit
                                    would run past the sequence's table pages     */
#define DAS_DEVERR_TESTED 8u     /* tested[b] outside [0, block_len]; clamped      */

/*
 * Depth-indexed, paged KV cache (caller-owned device memory).
 *
 * The cache stores, for each stored recurrence depth r ("plane"), each core
 * layer l and each KV head h, the verified prefix's K^{r,l} and V^{r,l}
 * (Sec. 2: depth-indexed cached representations; the core-layer index is
 * never remapped). Tokens live in pages of DAS_PAGE_TOKENS positions; a
 * sequence's logical page p is the physical page block_table[b][p], the same
 * physical page in every plane, layer and head.
 *
 *   k_pool: [num_k_planes][L][Hkv][num_pages][64][head_dim]     token-major
 *   v_pool: [num_v_planes][L][Hkv][num_pages][8][head_dim][8]   token-grouped
 *
 * Keys are stored token-major: position t of a page is row t. Values are
 * stored in groups of 8 positions: position t of a page is element
 * [t / 8][d][t % 8], so for every head dimension d the 8 positions of a
 * group are 16 contiguous bytes (bf16). Both products then read their
 * reduction dimension contiguously (Q K^T reduces over head_dim, P V over
 * positions), any 8-aligned run of positions of the value page is one
 * contiguous block, and a commit of 8 aligned positions writes one
 * contiguous head_dim x 16-byte block per (plane, layer, head).
 *
 * k_plane[r] / v_plane[r] (r = 1..R) give the plane holding depth r, or -1
 * when that depth is not stored; entry 0 is unused. Only the depths that a
 * workload reads need be stored.
 */
typedef struct das_cache {
  int32_t dtype;         /* das_dtype of every K/V/Q/O element               */
  int32_t num_depths;    /* R, 1..DAS_MAX_DEPTH                              */
  int32_t num_layers;    /* L core layers, >= 1                              */
  int32_t num_kv_heads;  /* Hkv, 1..65535                                    */
  int32_t head_dim;      /* 64, 96 or 128                                    */
  int32_t num_pages;     /* physical pages per (plane, layer, head), >= 1    */
  int32_t num_k_planes;  /* >= 1                                             */
  int32_t num_v_planes;  /* >= 1                                             */
  int32_t k_plane[DAS_MAX_DEPTH + 1];
  int32_t v_plane[DAS_MAX_DEPTH + 1];
  void *k_pool;
  void *v_pool;
} das_cache;

/*
 * A batch of sequences reading (or committing to) the cache.
 * prefix_len[b] is S_b, the number of verified, materialised positions of
 * sequence b (0 is legal). The anchor and the draft block are never prefix
 * positions. block_table has max_pages_per_seq columns; prefix_len[b] may
 * not exceed 64 * max_pages_per_seq. All three arrays are device memory.
 */
typedef struct das_batch {
  int32_t batch;               /* B, 1..65535                                 */
  int32_t max_pages_per_seq;   /* columns of block_table, 1..2^24, and
                                  batch * max_pages_per_seq < 2^31             */
  const int32_t *prefix_len;   /* device [B]                                  */
  const int32_t *block_table;  /* device [B][max_pages_per_seq], int32 pages  */
  uint32_t *dev_error;         /* optional device word (see DAS_DEVERR_*)     */
} das_batch;

/* Kernel family and schedule selection (measurement and tests). */
typedef enum das_attn_path {
  DAS_PATH_AUTO = 0,     /* library choice                                   */
  DAS_PATH_VALU = 1,     /* vector-ALU kernel (the only path for fp32)       */
  DAS_PATH_MFMA = 2,     /* matrix-core kernel over prefix splits (bf16)     */
  DAS_PATH_BALANCED = 3  /* matrix-core kernel, persistent balanced schedule:
                            every resident wave streams an equal share of
                            all sequences' tiles (bf16, 1..64 sequences,
                            blocks of at most 32 query rows, i.e.
                            w * Hq / Hkv <= 32, or 16 at head_dim 128;
                            DAS_ERR_UNSUPPORTED otherwise). DAS_PATH_AUTO takes it for batches
                            of 2..64 sequences when pages_per_split is 0
                            and the batch has more than W / 8 (sequence,
                            KV head) units, W = 256 x (7, 5, 4) workers
                            at head_dim (64, 96, 128). */
} das_attn_path;

typedef struct das_attn_options {
  int32_t path;             /* das_attn_path                                 */
  int32_t pages_per_split;  /* prefix pages per split (the first split of a
                               sequence, which also takes the draft block,
                               holds one page less); 0 = library choice;
                               clamped to the block table width + 1 (one
                               split then holds any sequence, and no merge
                               kernel runs), and to 64 on the matrix-core
                               path; not used by the balanced schedule      */
} das_attn_options;

/*
 * Bytes of device workspace an attention call with these shapes needs (the
 * partial results of the prefix splits or pieces: fp16 records with fp32
 * maxima and sums on the matrix-core paths, fp32 on the vector-ALU path).
 * Returns 0 for arguments that the attention entry points would reject.
 * `opts` may be NULL.
 */
size_t das_attn_workspace_bytes(const das_cache *cache, const das_batch *batch,
                                int32_t num_q_heads, int32_t block_len);
size_t das_attn_workspace_bytes_ex(const das_cache *cache, const das_batch *batch,
                                   int32_t num_q_heads, int32_t block_len,
                                   const das_attn_options *opts);

/*
 * Mature-V draft attention (Eq. (2)-(3) with the Mature-V / Deep V policy of
 * Eq. (4): kappa = draft_depth, nu = R). Prefix keys are read at the draft
 * depth d, prefix values at the full depth R, at core layer `layer`.
 *
 *   q      [B][w][Hq][head_dim]   queries of the current draft computation
 *   k_blk  [B][w][Hkv][head_dim]  draft-side keys at the current depth
 *   v_blk  [B][w][Hkv][head_dim]  draft-side values at the current depth
 *                                 (Mature-V changes prefix V only)
 *   out    [B][w][Hq][head_dim]   written, same dtype as the inputs
 *   lse    [B][Hq][w] fp32        optional natural-log softmax normaliser
 *   workspace                     >= das_attn_workspace_bytes(...) bytes,
 *                                 256-byte aligned, contents need no init;
 *                                 calls that run concurrently need separate
 *                                 workspaces
 *
 * w = block_len in 1..DAS_MAX_BLOCK; Hq a multiple of Hkv with Hq/Hkv <= 8;
 * layer in 0..L-1; draft_depth in 1..R; K at draft_depth and V at R stored.
 */
das_status das_attn_draft_maturev(const das_cache *cache, const das_batch *batch,
                                  int32_t layer, int32_t draft_depth,
                                  int32_t num_q_heads, int32_t block_len,
                                  const void *q, const void *k_blk, const void *v_blk,
                                  void *out, float *lse,
                                  void *workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/*
 * The target's ordinary attention at depth r (Aligned policy of Eq. (4),
 * kappa = nu = depth). With depth = R this is one core-layer attention of the
 * full-depth verifier of Sec. 3.4, over the verifier input block
 * [x_t, y_1 .. y_{w-1}]. Arguments as for das_attn_draft_maturev, with the
 * block tensors at depth `depth`.
 */
das_status das_attn_verify(const das_cache *cache, const das_batch *batch,
                           int32_t layer, int32_t depth,
                           int32_t num_q_heads, int32_t block_len,
                           const void *q, const void *k_blk, const void *v_blk,
                           void *out, float *lse,
                           void *workspace, size_t workspace_bytes,
                           hipStream_t stream);

/*
 * Any read policy of Eq. (4): prefix keys at depth kappa, prefix values at
 * depth nu (Aligned (r,r), Mature-V (r,R), Deep K (R,r), Deep K/V (R,R)).
 * The two entry points above are this call with fixed (kappa, nu).
 * `opts` may be NULL (library choices); a workspace sized with the same
 * `opts` must be passed.
 */
das_status das_attn_policy(const das_cache *cache, const das_batch *batch,
                           int32_t layer, int32_t kappa, int32_t nu,
                           int32_t num_q_heads, int32_t block_len,
                           const void *q, const void *k_blk, const void *v_blk,
                           void *out, float *lse,
                           void *workspace, size_t workspace_bytes,
                           const das_attn_options *opts, hipStream_t stream);

/* Bytes of the library-owned scratch of das_attn_policy_noalloc (per GPU). */
#define DAS_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * das_attn_policy without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation). The split partials go to a
 * library-owned scratch array of DAS_NOALLOC_SCRATCH_BYTES bytes per GPU,
 * placed when the library's code is loaded on that GPU and held until the
 * process ends; this call allocates nothing. Results are those of
 * das_attn_policy with the same arguments and `opts`, bit for bit.
 *
 * - The first call on a device (with that device current) looks up the
 *   device address of that device's scratch copy; `stream` must belong to
 *   the current device (DAS_ERR_UNSUPPORTED otherwise; NULL = the current
 *   device's null stream).
 * - DAS_ERR_WORKSPACE when the request's workspace
 *   (das_attn_workspace_bytes_ex with the same arguments) exceeds
 *   DAS_NOALLOC_SCRATCH_BYTES.
 * - Every call on a GPU shares that GPU's scratch, and the scratch keeps
 *   whatever the last call left there (nothing in it needs clearing: each
 *   call writes every partial it reads). Calls that can overlap on one GPU
 *   (on different streams, or from different threads without ordering)
 *   race on it: serialise them on one stream, or use das_attn_policy with
 *   separate workspaces.
 */
das_status das_attn_policy_noalloc(const das_cache *cache, const das_batch *batch,
                                   int32_t layer, int32_t kappa, int32_t nu,
                                   int32_t num_q_heads, int32_t block_len,
                                   const void *q, const void *k_blk, const void *v_blk,
                                   void *out, float *lse, const das_attn_options *opts,
                                   hipStream_t stream);

/*
 * Commit (Sec. 3.4; App. B.1): for each sequence b, write the full-depth K/V
 * of the first num_new[b] block inputs to prefix positions
 * prefix_len[b] .. prefix_len[b] + num_new[b] - 1, in every stored plane and
 * every core layer. Entries past num_new[b] (rejected candidates) are not
 * written. Draft-side K/V are never committed.
 *
 *   k_new   [num_k_planes][L][B][w_max][Hkv][head_dim]  plane order = k_pool
 *   v_new   [num_v_planes][L][B][w_max][Hkv][head_dim]  plane order = v_pool
 *   num_new device [B] int32, each in 0..w_max
 *   len_out device [B] int32 or NULL: receives prefix_len[b] + num_new[b];
 *           must not alias batch->prefix_len
 *
 * The target pages must already be present in block_table. The verifier's
 * block K/V at plane p and layer l, k_new[p][l], is the same buffer the
 * attention calls take as k_blk. DAS_ERR_SHAPE when w_max is outside
 * 1..DAS_MAX_BLOCK or the commit's grid (one 64-lane wave per (plane, layer,
 * KV head), four per workgroup) exceeds 2^32 - 1 work-items.
 */
das_status das_kv_append(const das_cache *cache, const das_batch *batch,
                         const void *k_new, const void *v_new, int32_t w_max,
                         const int32_t *num_new, int32_t *len_out,
                         hipStream_t stream);

/*
 * Greedy verification of a block on the device (Sec. 3.4), so that the
 * commit count reaches das_kv_append without a host round trip.
 *
 * For each sequence b, the first m_b = tested[b] proposals are checked in
 * order against the verifier's predictions; proposals are accepted while
 * y_i equals yhat_i (i = 1..m_b). With a_b accepted:
 *   - emitted tokens: y_1..y_{a_b}, then yhat_{a_b+1} when a_b < w (the
 *     target prediction at the first mismatch, or the bonus token from an
 *     unused conditional when all m_b < w tested proposals agree); w tokens
 *     when every proposal of a full block is accepted;
 *   - retained verifier inputs: num_keep[b] = min(a_b + 1, w) (the anchor and
 *     the accepted inputs among [x_t, y_1 .. y_{w-1}]).
 *
 *   proposals   device [B][w] int32: y_1..y_w (index i-1 holds y_i)
 *   target_pred device [B][w] int32: yhat_i = argmax of the verifier's
 *               conditional p_i (computed by the model's readout)
 *   tested      device [B] int32 m_b in 0..w, or NULL for m_b = w; values
 *               outside 0..w are clamped and reported with DAS_DEVERR_TESTED
 *   accepted    device [B] int32, written: a_b
 *   num_keep    device [B] int32, written: min(a_b + 1, w); pass it as the
 *               num_new argument of das_kv_append (w_max = w)
 *   emitted     device [B][w] int32 or NULL, written: the emitted tokens;
 *               entries past num_emitted[b] are left untouched
 *   num_emitted device [B] int32 or NULL, written: min(a_b + 1, w)
 *   dev_error   optional device word (DAS_DEVERR_TESTED)
 *
 * batch >= 1; block_len w in 1..DAS_MAX_BLOCK. Integer work only: results
 * are exact. The output arrays must not overlap the inputs.
 */
das_status das_greedy_accept(int32_t batch, int32_t block_len, const int32_t *proposals,
                             const int32_t *target_pred, const int32_t *tested,
                             int32_t *accepted, int32_t *num_keep, int32_t *emitted,
                             int32_t *num_emitted, uint32_t *dev_error, hipStream_t stream);

/* Static description of a status code; never NULL. */
const char *das_status_string(das_status status);

/* Library version as major * 10000 + minor * 100 + patch. */
int32_t das_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DAS_H */
