// Host side of the DAS attention library: argument validation, split
// planning, workspace sizing and kernel dispatch behind the C ABI of das.h.
//
// Every check runs before the first HIP call, so a rejected request has
// enqueued nothing and the checks can be exercised without a GPU.

#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "das_internal.h"

namespace das {
namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int elem_bytes(int dtype) { return dtype == DAS_F32 ? 4 : 2; }

bool aligned(const void *ptr, size_t a) { return reinterpret_cast<uintptr_t>(ptr) % a == 0; }

das_status check_cache(const das_cache *c) {
  if (!c) return DAS_ERR_NULL;
  if (!c->k_pool || !c->v_pool) return DAS_ERR_NULL;
  if (!aligned(c->k_pool, 16) || !aligned(c->v_pool, 16)) return DAS_ERR_ALIGN;
  if (c->dtype != DAS_F32 && c->dtype != DAS_BF16) return DAS_ERR_DTYPE;
  if (c->num_depths < 1 || c->num_depths > DAS_MAX_DEPTH) return DAS_ERR_SHAPE;
  if (c->num_layers < 1 || c->num_kv_heads < 1 || c->num_pages < 1) return DAS_ERR_SHAPE;
  if (c->num_kv_heads > 65535) return DAS_ERR_SHAPE;
  if (c->num_k_planes < 1 || c->num_v_planes < 1) return DAS_ERR_SHAPE;
  if (c->head_dim != 64 && c->head_dim != 96 && c->head_dim != 128) return DAS_ERR_SHAPE;
  for (int r = 1; r <= c->num_depths; ++r) {
    if (c->k_plane[r] < -1 || c->k_plane[r] >= c->num_k_planes) return DAS_ERR_SHAPE;
    if (c->v_plane[r] < -1 || c->v_plane[r] >= c->num_v_planes) return DAS_ERR_SHAPE;
  }
  return DAS_OK;
}

das_status check_batch(const das_batch *b) {
  if (!b) return DAS_ERR_NULL;
  if (!b->prefix_len || !b->block_table) return DAS_ERR_NULL;
  if (!aligned(b->prefix_len, 4) || !aligned(b->block_table, 4) || !aligned(b->dev_error, 4))
    return DAS_ERR_ALIGN;
  if (b->batch < 1 || b->batch > 65535 || b->max_pages_per_seq < 1) return DAS_ERR_SHAPE;
  // positions (pages x 64) and table offsets (B x pages) stay within int32
  if (b->max_pages_per_seq > (1 << 24) ||
      static_cast<long long>(b->batch) * b->max_pages_per_seq > 0x7fffffffLL)
    return DAS_ERR_SHAPE;
  return DAS_OK;
}

// Which kernel family (and schedule) runs a request. The balanced schedule
// serves batches with many (sequence, KV head) units: every resident wave
// streams an equal share of all tiles, so unequal prefix lengths leave no
// idle slots. With few units for the chip's workers (at most 8 workers per
// unit) each worker holds a short run behind its dependent start-up round
// trips and leaves one piece per unit it shares, and the split grid's
// chunks, dealt out by the hardware dispatcher, are faster; a single
// sequence has nothing to balance and keeps the split grid too.
bool balanced_pays(const das_cache *c, const das_batch *b) {
  return 8LL * b->batch * c->num_kv_heads >
         static_cast<long long>(kNumCUs) * balanced_workers_per_cu(c->head_dim);
}

int choose_path(const das_cache *c, const das_batch *b, int rows, const das_attn_options *o) {
  const int want = o ? o->path : DAS_PATH_AUTO;
  if (c->dtype == DAS_F32) return DAS_PATH_VALU;
  if (want != DAS_PATH_AUTO) return want;
  if (b->batch >= 2 && b->batch <= kBalancedMaxBatch && rows <= balanced_max_rows(c->head_dim) &&
      !(o && o->pages_per_split != 0) && balanced_pays(c, b))
    return DAS_PATH_BALANCED;
  return DAS_PATH_MFMA;
}

struct Plan {
  int path;
  int rows;             // w * G query rows per (sequence, kv head)
  int pages_per_split;
  int nsplit;
  int nsplit_ml;        // nsplit rounded up to a multiple of 4
  int n_workers;        // balanced schedule: workers launched
  int piece_cap;        // balanced schedule: pieces the workspace holds
  int piece_stride;     // matrix-core kernels: bytes of one piece record
  size_t ws_o_bytes, ws_ml_bytes, ws_rec_bytes, total;
};

// Prefix pages of one sequence are cut into splits of pages_per_split pages;
// each (split, KV head, row tile) is one chunk of work, one workgroup. The
// default aims for at least ~1024 chunks (four single-wave workgroups per
// compute unit of a 256-CU part): with `units` = sequences x KV heads x row
// tiles, each (sequence, KV head) gets max(2, the largest power of two
// <= 1024 / units) splits, and a split holds between 2 and 32 pages.
// (Measured on MI355X over 1-64 pages per split on the single-sequence,
// ragged, long-prefix and wave-step workloads: this picks the best split
// size on three and one within 0.5 % of the best on the fourth.)
das_status make_plan(const das_cache *c, const das_batch *b, int hq, int w,
                     const das_attn_options *o, Plan *plan) {
  if (hq < 1 || hq % c->num_kv_heads != 0) return DAS_ERR_SHAPE;
  const int group = hq / c->num_kv_heads;
  if (group > 8) return DAS_ERR_UNSUPPORTED;
  if (w < 1 || w > DAS_MAX_BLOCK) return DAS_ERR_SHAPE;
  if (o && (o->pages_per_split < 0 || o->path < DAS_PATH_AUTO || o->path > DAS_PATH_BALANCED))
    return DAS_ERR_SHAPE;
  if (o && (o->path == DAS_PATH_MFMA || o->path == DAS_PATH_BALANCED) && c->dtype != DAS_BF16)
    return DAS_ERR_UNSUPPORTED;
  plan->rows = w * group;
  plan->path = choose_path(c, b, plan->rows, o);
  if (plan->path == DAS_PATH_BALANCED) {
    if (b->batch > kBalancedMaxBatch || plan->rows > balanced_max_rows(c->head_dim))
      return DAS_ERR_UNSUPPORTED;
    // workers: one per resident single-wave workgroup of the chip; pieces:
    // at most units + workers - 1 (index unit + worker)
    plan->n_workers = kNumCUs * balanced_workers_per_cu(c->head_dim);
    plan->piece_cap = b->batch * c->num_kv_heads + plan->n_workers;
    plan->pages_per_split = 0;
    plan->nsplit = 0;
    plan->nsplit_ml = 0;
    // a piece record: the rows' fp16 outputs, then 16 bytes per row
    plan->piece_stride = static_cast<int>(piece_record_bytes(plan->rows, c->head_dim));
    const size_t pieces = static_cast<size_t>(plan->piece_cap);
    plan->ws_o_bytes = pieces * plan->piece_stride;
    plan->ws_ml_bytes = 0;
    plan->ws_rec_bytes =
        align_up(static_cast<size_t>(b->batch) * c->num_kv_heads * 2 * sizeof(int32_t));
    plan->total = plan->ws_o_bytes + plan->ws_rec_bytes;
    // merge grid: (sequence, KV head) x 64 threads along x
    if (static_cast<long long>(b->batch) * c->num_kv_heads * 64 > 0xffffffffLL)
      return DAS_ERR_SHAPE;
    return DAS_OK;
  }
  plan->n_workers = 0;
  plan->piece_cap = 0;
  plan->piece_stride = 0;
  plan->ws_rec_bytes = 0;
  const int maxp = b->max_pages_per_seq;
  int pps = o ? o->pages_per_split : 0;
  if (pps == 0) {
    const long tile_rows = plan->path == DAS_PATH_MFMA ? (plan->rows <= 16 ? 16 : 32)
                                                      : valu_tile_rows(plan->rows);
    const long units = static_cast<long>(b->batch) * c->num_kv_heads *
                       ((plan->rows + tile_rows - 1) / tile_rows);
    // about two chunks per CU: longer chunks amortise their first round
    // trip and leave fewer partials to merge. Matrix-core blocks of more than
    // 32 rows run their row tiles as the waves of one workgroup (two per CU):
    // they take four times the row-tile chunks. On the vector-ALU path a
    // split may be one page.
    const bool mfma = plan->path == DAS_PATH_MFMA;
    const long target = mfma && plan->rows > 32 ? 2048 : 512;
    long splits = 2;
    while (splits * 2 * units <= target) splits *= 2;
    long want = maxp / splits;
    if (want < (mfma ? 2 : 1)) want = mfma ? 2 : 1;
    if (want > 32) want = 32;
    pps = static_cast<int>(want);
  }
  // at most maxp + 1 pages: one split then holds any sequence and its block
  if (pps > maxp + 1) pps = maxp + 1;
  if (plan->path == DAS_PATH_MFMA && pps > kMaxPagesPerSplit) pps = kMaxPagesPerSplit;
  plan->pages_per_split = pps;
  plan->nsplit = splits_of(maxp, pps);
  // Every grid dimension of the launches stays within what HIP accepts:
  // at most 2^32 - 1 work-items (workgroups x threads) per dimension.
  const long long kMaxItems = 0xffffffffLL;
  const long long units = static_cast<long long>(b->batch) * c->num_kv_heads;
  if (plan->path == DAS_PATH_MFMA) {
    const long long nq = mfma_tiles_per_wave(plan->rows), nw = mfma_waves(plan->rows);
    const long long n_rt = (plan->rows + 16 * nq - 1) / (16 * nq);
    const long long chunks = units * plan->nsplit * ((n_rt + nw - 1) / nw);
    if (chunks * 64 * nw > kMaxItems) return DAS_ERR_SHAPE;
  } else {
    const long long n_rt = (plan->rows + valu_tile_rows(plan->rows) - 1) /
                           valu_tile_rows(plan->rows);
    // grid (splits, KV heads, sequences x row tiles) of 256-thread workgroups
    if (static_cast<long long>(plan->nsplit) * 256 > kMaxItems ||
        static_cast<long long>(b->batch) * n_rt > 65535)
      return DAS_ERR_SHAPE;
  }
  if (units * 64 > kMaxItems) return DAS_ERR_SHAPE;  // the merge: (sequence, KV head) x 64
  plan->nsplit_ml = (plan->nsplit + 3) & ~3;
  if (plan->path == DAS_PATH_MFMA) {
    // one piece record per (sequence, KV head, split)
    plan->piece_stride = static_cast<int>(piece_record_bytes(plan->rows, c->head_dim));
    plan->ws_o_bytes = static_cast<size_t>(units) * plan->nsplit * plan->piece_stride;
    plan->ws_ml_bytes = 0;
    plan->total = plan->ws_o_bytes;
    return DAS_OK;
  }
  const size_t per_split_rows =
      static_cast<size_t>(b->batch) * c->num_kv_heads * plan->nsplit * plan->rows;
  plan->ws_o_bytes = align_up(per_split_rows * c->head_dim * sizeof(float));
  plan->ws_ml_bytes = align_up(static_cast<size_t>(b->batch) * c->num_kv_heads * plan->rows *
                               plan->nsplit_ml * sizeof(float));
  plan->total = plan->ws_o_bytes + 2 * plan->ws_ml_bytes;
  return DAS_OK;
}

// Validates an attention request and fills every launch parameter except the
// workspace pointers. No HIP call.
das_status prepare_attn(const das_cache *c, const das_batch *b, int layer, int kappa, int nu,
                        int hq, int w, const void *q, const void *kb, const void *vb,
                        void *out, float *lse, const das_attn_options *o, AttnParams *pp,
                        Plan *plan) {
  das_status st = check_cache(c);
  if (st != DAS_OK) return st;
  st = check_batch(b);
  if (st != DAS_OK) return st;
  if (!q || !kb || !vb || !out) return DAS_ERR_NULL;
  if (!aligned(q, 16) || !aligned(kb, 16) || !aligned(vb, 16) || !aligned(out, 16) ||
      !aligned(lse, 4))
    return DAS_ERR_ALIGN;
  if (layer < 0 || layer >= c->num_layers) return DAS_ERR_SHAPE;
  if (kappa < 1 || kappa > c->num_depths || nu < 1 || nu > c->num_depths) return DAS_ERR_DEPTH;
  const int kplane = c->k_plane[kappa];
  const int vplane = c->v_plane[nu];
  if (kplane < 0 || vplane < 0) return DAS_ERR_DEPTH;
  st = make_plan(c, b, hq, w, o, plan);
  if (st != DAS_OK) return st;

  const int dh = c->head_dim;
  const size_t eb = static_cast<size_t>(elem_bytes(c->dtype));
  const size_t layer_elems = static_cast<size_t>(c->num_kv_heads) * c->num_pages * kPage * dh;
  AttnParams &p = *pp;
  p.k_layer = static_cast<const char *>(c->k_pool) +
              (static_cast<size_t>(kplane) * c->num_layers + layer) * layer_elems * eb;
  p.v_layer = static_cast<const char *>(c->v_pool) +
              (static_cast<size_t>(vplane) * c->num_layers + layer) * layer_elems * eb;
  p.q = q;
  p.kb = kb;
  p.vb = vb;
  p.out = out;
  p.lse = lse;
  p.prefix_len = b->prefix_len;
  p.block_table = b->block_table;
  p.dev_error = b->dev_error;
  p.ws_o = p.ws_m = p.ws_l = nullptr;
  p.ws_rec = nullptr;
  p.batch = b->batch;
  p.hq = hq;
  p.hkv = c->num_kv_heads;
  p.group = hq / c->num_kv_heads;
  p.w = w;
  p.rows = plan->rows;
  p.num_pages = c->num_pages;
  p.max_pages = b->max_pages_per_seq;
  p.pages_per_split = plan->pages_per_split;
  p.nsplit = plan->nsplit;
  p.nsplit_ml = plan->nsplit_ml;
  p.n_workers = plan->n_workers;
  p.piece_cap = plan->piece_cap;
  p.piece_stride = plan->piece_stride;
  // log2(e) / sqrt(dh): logits are kept in base-2 units so exp2 can be used.
  const double log2e = 1.4426950408889634074;
  p.scale_log2 = static_cast<float>(log2e / __builtin_sqrt(static_cast<double>(dh)));
  return DAS_OK;
}

// Enqueues a prepared request with its workspace (plan.total bytes at ws,
// 256-byte aligned): the attention kernel, then the split merge when a
// sequence can span several splits.
das_status launch_attn(AttnParams p, const Plan &plan, int dtype, int dh, void *ws,
                       hipStream_t stream) {
  char *wsb = static_cast<char *>(ws);
  p.ws_o = reinterpret_cast<float *>(wsb);
  p.ws_m = reinterpret_cast<float *>(wsb + plan.ws_o_bytes);
  p.ws_l = reinterpret_cast<float *>(wsb + plan.ws_o_bytes + plan.ws_ml_bytes);
  p.ws_rec = reinterpret_cast<int32_t *>(wsb + plan.ws_o_bytes + 2 * plan.ws_ml_bytes);
  if (plan.path == DAS_PATH_BALANCED)
    return launch_attn_balanced(p, dh, stream) == hipSuccess ? DAS_OK : DAS_ERR_HIP;
  const bool mfma = plan.path == DAS_PATH_MFMA;
  const hipError_t e = mfma ? launch_attn_mfma(p, dh, stream)
                            : launch_attn_valu(p, dtype, dh, stream);
  if (e != hipSuccess) return DAS_ERR_HIP;
  // one split per sequence: the attention kernel wrote every output itself
  if (plan.nsplit > 1 && (mfma ? launch_attn_combine_records(p, dh, 1, stream)
                              : launch_attn_combine(p, dtype, dh, 1, stream)) != hipSuccess)
    return DAS_ERR_HIP;
  return DAS_OK;
}

das_status attn_common(const das_cache *c, const das_batch *b, int layer, int kappa, int nu,
                       int hq, int w, const void *q, const void *kb, const void *vb, void *out,
                       float *lse, void *ws, size_t ws_bytes, const das_attn_options *o,
                       hipStream_t stream) {
  AttnParams p;
  Plan plan;
  const das_status st = prepare_attn(c, b, layer, kappa, nu, hq, w, q, kb, vb, out, lse, o,
                                     &p, &plan);
  if (st != DAS_OK) return st;
  if (!ws || ws_bytes < plan.total) return DAS_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0) return DAS_ERR_WORKSPACE;
  return launch_attn(p, plan, c->dtype, c->head_dim, ws, stream);
}

// ---------------------------------------------------------------------------
// Library-owned scratch of the allocation-free attention entry point: one
// copy per GPU, part of the code object (the loader places it when the
// library's code is loaded on a device, and it lives until the process ends).
// Host code never passes `scratch` itself to a kernel (in host code the name
// stands for a host-side shadow, not a device address): the device address of
// each GPU's copy is looked up once per device with hipGetSymbolAddress, with
// that device current, and kept in scratch_ptr[].
// ---------------------------------------------------------------------------
constexpr int kMaxDevices = 64;
__device__ __attribute__((aligned(256))) uint8_t scratch[DAS_NOALLOC_SCRATCH_BYTES];
void *scratch_ptr[kMaxDevices];
std::mutex scratch_mutex;

// Device address of the current device's scratch copy, or nullptr.
void *scratch_of_current_device(das_status *st) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    *st = DAS_ERR_HIP;
    return nullptr;
  }
  if (dev >= kMaxDevices) {
    *st = DAS_ERR_UNSUPPORTED;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      *st = DAS_ERR_HIP;
      return nullptr;
    }
    scratch_ptr[dev] = ptr;
  }
  return scratch_ptr[dev];
}

}  // namespace
}  // namespace das

using namespace das;

extern "C" {

size_t das_attn_workspace_bytes_ex(const das_cache *cache, const das_batch *batch,
                                   int32_t num_q_heads, int32_t block_len,
                                   const das_attn_options *opts) {
  if (check_cache(cache) != DAS_OK || check_batch(batch) != DAS_OK) return 0;
  Plan plan;
  if (make_plan(cache, batch, num_q_heads, block_len, opts, &plan) != DAS_OK) return 0;
  return plan.total;
}

size_t das_attn_workspace_bytes(const das_cache *cache, const das_batch *batch,
                                int32_t num_q_heads, int32_t block_len) {
  return das_attn_workspace_bytes_ex(cache, batch, num_q_heads, block_len, nullptr);
}

das_status das_attn_policy(const das_cache *cache, const das_batch *batch, int32_t layer,
                           int32_t kappa, int32_t nu, int32_t num_q_heads, int32_t block_len,
                           const void *q, const void *k_blk, const void *v_blk, void *out,
                           float *lse, void *workspace, size_t workspace_bytes,
                           const das_attn_options *opts, hipStream_t stream) {
  return attn_common(cache, batch, layer, kappa, nu, num_q_heads, block_len, q, k_blk, v_blk,
                     out, lse, workspace, workspace_bytes, opts, stream);
}

das_status das_attn_policy_noalloc(const das_cache *cache, const das_batch *batch,
                                   int32_t layer, int32_t kappa, int32_t nu,
                                   int32_t num_q_heads, int32_t block_len, const void *q,
                                   const void *k_blk, const void *v_blk, void *out, float *lse,
                                   const das_attn_options *opts, hipStream_t stream) {
  AttnParams p;
  Plan plan;
  das_status st = prepare_attn(cache, batch, layer, kappa, nu, num_q_heads, block_len, q,
                               k_blk, v_blk, out, lse, opts, &p, &plan);
  if (st != DAS_OK) return st;
  if (plan.total > DAS_NOALLOC_SCRATCH_BYTES) return DAS_ERR_WORKSPACE;
  // the stream must belong to the current device, whose scratch copy is used
  if (stream) {
    int cur = -1, sdev = -1;
    if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(stream, &sdev) != hipSuccess)
      return DAS_ERR_HIP;
    if (sdev != cur) return DAS_ERR_UNSUPPORTED;
  }
  void *ws = scratch_of_current_device(&st);
  if (!ws) return st;
  return launch_attn(p, plan, cache->dtype, cache->head_dim, ws, stream);
}

das_status das_attn_draft_maturev(const das_cache *cache, const das_batch *batch,
                                  int32_t layer, int32_t draft_depth, int32_t num_q_heads,
                                  int32_t block_len, const void *q, const void *k_blk,
                                  const void *v_blk, void *out, float *lse, void *workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  if (!cache) return DAS_ERR_NULL;
  // Mature-V: keys at the draft depth, values at the full depth R.
  return attn_common(cache, batch, layer, draft_depth, cache->num_depths, num_q_heads,
                     block_len, q, k_blk, v_blk, out, lse, workspace, workspace_bytes,
                     nullptr, stream);
}

das_status das_attn_verify(const das_cache *cache, const das_batch *batch, int32_t layer,
                           int32_t depth, int32_t num_q_heads, int32_t block_len,
                           const void *q, const void *k_blk, const void *v_blk, void *out,
                           float *lse, void *workspace, size_t workspace_bytes,
                           hipStream_t stream) {
  // Aligned read: keys and values at the same depth.
  return attn_common(cache, batch, layer, depth, depth, num_q_heads, block_len, q, k_blk,
                     v_blk, out, lse, workspace, workspace_bytes, nullptr, stream);
}

das_status das_kv_append(const das_cache *cache, const das_batch *batch, const void *k_new,
                         const void *v_new, int32_t w_max, const int32_t *num_new,
                         int32_t *len_out, hipStream_t stream) {
  das_status st = check_cache(cache);
  if (st != DAS_OK) return st;
  st = check_batch(batch);
  if (st != DAS_OK) return st;
  if (!k_new || !v_new || !num_new) return DAS_ERR_NULL;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(num_new, 4) ||
      !aligned(len_out, 4))
    return DAS_ERR_ALIGN;
  if (w_max < 1 || w_max > DAS_MAX_BLOCK) return DAS_ERR_SHAPE;
  // The commit's grid: one wave per (plane, layer, KV head), four per
  // 256-thread workgroup, keys and values in separate workgroups; at most
  // 2^32 - 1 work-items along x.
  const long long per_plane = static_cast<long long>(cache->num_layers) * cache->num_kv_heads;
  const long long blocks = (cache->num_k_planes * per_plane + 3) / 4 +
                           (cache->num_v_planes * per_plane + 3) / 4;
  if (blocks * 256 > 0xffffffffLL) return DAS_ERR_SHAPE;
  if (len_out && static_cast<const void *>(len_out) ==
                     static_cast<const void *>(batch->prefix_len))
    return DAS_ERR_SHAPE;
  AppendParams p;
  p.k_new = k_new;
  p.v_new = v_new;
  p.k_pool = cache->k_pool;
  p.v_pool = cache->v_pool;
  p.prefix_len = batch->prefix_len;
  p.block_table = batch->block_table;
  p.num_new = num_new;
  p.len_out = len_out;
  p.dev_error = batch->dev_error;
  p.batch = batch->batch;
  p.n_k_planes = cache->num_k_planes;
  p.n_v_planes = cache->num_v_planes;
  p.layers = cache->num_layers;
  p.hkv = cache->num_kv_heads;
  p.num_pages = cache->num_pages;
  p.max_pages = batch->max_pages_per_seq;
  p.w_max = w_max;
  if (launch_kv_append(p, cache->dtype, cache->head_dim, stream) != hipSuccess)
    return DAS_ERR_HIP;
  return DAS_OK;
}

das_status das_greedy_accept(int32_t batch, int32_t block_len, const int32_t *proposals,
                             const int32_t *target_pred, const int32_t *tested,
                             int32_t *accepted, int32_t *num_keep, int32_t *emitted,
                             int32_t *num_emitted, uint32_t *dev_error, hipStream_t stream) {
  if (!proposals || !target_pred || !accepted || !num_keep) return DAS_ERR_NULL;
  if (batch < 1 || block_len < 1 || block_len > DAS_MAX_BLOCK) return DAS_ERR_SHAPE;
  if (!aligned(proposals, 4) || !aligned(target_pred, 4) || !aligned(tested, 4) ||
      !aligned(accepted, 4) || !aligned(num_keep, 4) || !aligned(emitted, 4) ||
      !aligned(num_emitted, 4) || !aligned(dev_error, 4))
    return DAS_ERR_ALIGN;
  AcceptParams p;
  p.proposals = proposals;
  p.target_pred = target_pred;
  p.tested = tested;
  p.accepted = accepted;
  p.num_keep = num_keep;
  p.emitted = emitted;
  p.num_emitted = num_emitted;
  p.dev_error = dev_error;
  p.batch = batch;
  p.w = block_len;
  if (launch_greedy_accept(p, stream) != hipSuccess) return DAS_ERR_HIP;
  return DAS_OK;
}

const char *das_status_string(das_status status) {
  switch (status) {
    case DAS_OK: return "ok";
    case DAS_ERR_NULL: return "a required pointer is NULL";
    case DAS_ERR_SHAPE: return "a size is out of range or inconsistent";
    case DAS_ERR_DEPTH: return "depth outside 1..R or not stored in the cache";
    case DAS_ERR_DTYPE: return "unknown element type";
    case DAS_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case DAS_ERR_HIP: return "a HIP kernel launch failed";
    case DAS_ERR_UNSUPPORTED: return "request not supported by this build";
    case DAS_ERR_ALIGN: return "a device array is not aligned as required";
  }
  return "unknown status";
}

int32_t das_version(void) { return 100; }

}  // extern "C"
