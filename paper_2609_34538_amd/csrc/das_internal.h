// Internal declarations shared by the host dispatcher and the kernels of the
// DAS attention library. Not part of the public C ABI (include/das.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "das.h"

namespace das {

constexpr int kPage = DAS_PAGE_TOKENS;  // tokens per cache page
constexpr int kMaxPagesPerSplit = 64;   // matrix-core kernel: one page id per lane

// Everything one attention launch needs. Pointers are device pointers; the
// pool pointers already include the plane and core-layer offsets, so a
// kernel only adds (kv head, page) offsets.
struct AttnParams {
  const void *k_layer;   // [Hkv][P][64][dh]   keys of plane kappa, layer l
  const void *v_layer;   // [Hkv][P][8][dh][8] values of plane nu, layer l
  const void *q;         // [B][w][Hq][dh]
  const void *kb;        // [B][w][Hkv][dh]
  const void *vb;        // [B][w][Hkv][dh]
  void *out;             // [B][w][Hq][dh]
  float *lse;            // [B][Hq][w] or nullptr
  const int32_t *prefix_len;   // [B]
  const int32_t *block_table;  // [B][max_pages]
  uint32_t *dev_error;         // or nullptr
  float *ws_o;           // [B][Hkv][nsplit][rows][dh]     unnormalised partial O
                         // (matrix-core kernels: piece records, see piece_stride)
  float *ws_m;           // [B][Hkv][rows][nsplit_ml]      running max (log2 units)
  float *ws_l;           // [B][Hkv][rows][nsplit_ml]      running sum
  int32_t batch, hq, hkv, group, w, rows;  // rows = w * group
  int32_t num_pages, max_pages;
  int32_t pages_per_split, nsplit;
  int32_t nsplit_ml;     // nsplit rounded up to a multiple of 4 (16-byte rows of m, l)
  float scale_log2;      // log2(e) / sqrt(dh): logits in base-2 units
  // balanced schedule only: workers launched (one single-wave workgroup
  // each) and the piece capacity of the workspace
  int32_t n_workers, piece_cap;
  // matrix-core kernels: bytes of one piece record at ws_o
  // (piece_record_bytes; split grid: record (b * Hkv + kvh) * nsplit + split)
  int32_t piece_stride;
  int32_t *ws_rec;       // balanced schedule: per unit {first piece, piece count}
};

struct AppendParams {
  const void *k_new;     // [nK][L][B][w_max][Hkv][dh]
  const void *v_new;     // [nV][L][B][w_max][Hkv][dh]
  void *k_pool;          // [nK][L][Hkv][P][64][dh]
  void *v_pool;          // [nV][L][Hkv][P][8][dh][8]
  const int32_t *prefix_len;
  const int32_t *block_table;
  const int32_t *num_new;
  int32_t *len_out;
  uint32_t *dev_error;
  int32_t batch, n_k_planes, n_v_planes, layers, hkv, num_pages, max_pages, w_max;
};

template <typename... KArgs>
hipError_t launch_kernel_impl(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s,
                              KArgs... args) {
  void *argv[] = {static_cast<void *>(&args)...};
  return hipLaunchKernel(reinterpret_cast<const void *>(kernel), grid, block, argv, 0, s);
}

// Enqueues kernel<<<grid, block, 0, s>>>(args...) and returns the status of
// that launch alone: hipLaunchKernel reports it directly, so an error left
// pending by the caller's earlier HIP work is neither taken for this launch's
// nor cleared.
template <typename... KArgs, typename... Args>
hipError_t launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t s,
                         Args &&...args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
  return launch_kernel_impl<KArgs...>(kernel, grid, block, s, static_cast<KArgs>(args)...);
}

// Launchers (return the hipError_t of the launch).
hipError_t launch_attn_valu(const AttnParams &p, int dtype, int dh, hipStream_t s);
hipError_t launch_attn_mfma(const AttnParams &p, int dh, hipStream_t s);
// skip_single: sequences whose prefix fits one split were already written
// by the attention kernel (both kernel families write them directly).
hipError_t launch_attn_combine(const AttnParams &p, int dtype, int dh, int skip_single,
                               hipStream_t s);
// The same over the piece records the matrix-core kernel writes (bf16 output).
hipError_t launch_attn_combine_records(const AttnParams &p, int dh, int skip_single,
                                       hipStream_t s);
hipError_t launch_kv_append(const AppendParams &p, int dtype, int dh, hipStream_t s);
// Balanced persistent schedule for batches of up to 64 sequences with blocks
// of at most balanced_max_rows(dh) query rows (bf16): the attention kernel
// and its piece merge.
hipError_t launch_attn_balanced(const AttnParams &p, int dh, hipStream_t s);
constexpr int kBalancedMaxBatch = 64;
// query rows per (sequence, KV head) the balanced kernel takes
__host__ __device__ constexpr int balanced_max_rows(int dh) { return dh == 128 ? 16 : 32; }
// Bytes of one piece record of the matrix-core kernels (a partial result
// over part of a unit's positions): [rows][dh] fp16 outputs, then 16 bytes
// per row, 256-byte aligned.
__host__ __device__ constexpr size_t piece_record_bytes(int rows, int dh) {
  return (static_cast<size_t>(rows) * (2 * dh + 16) + 255) / 256 * 256;
}
constexpr int kNumCUs = 256;  // compute units of an MI355X (gfx950)
// Workers of the balanced schedule per compute unit: 64 KB of tiles in flight
// per CU, one 128 * dh-byte tile per worker, as long as every worker's LDS
// (two ring slots and one stashed piece record) fits strictly inside the
// 160 KB: 7 at head dim 64, 5 at 96, 4 at 128. Measured against the workers
// whose rings alone fill the LDS (10, 6, 5): 0.78 against 0.63, 0.78 against
// 0.78 and 0.80 against 0.60 of 8 TB/s on the DAS-Wave step's shape at each
// head dim; when the LDS is filled exactly (head dims 64 and 128) a CU's
// last worker is not resident with the others and runs after them.
__host__ __device__ constexpr int balanced_lds_per_worker(int dh) {
  return 2 * 128 * dh + static_cast<int>(piece_record_bytes(balanced_max_rows(dh), dh));
}
__host__ __device__ constexpr int balanced_workers_per_cu(int dh) {
  return 512 / dh < (160 * 1024 - 1) / balanced_lds_per_worker(dh)
             ? 512 / dh
             : (160 * 1024 - 1) / balanced_lds_per_worker(dh);
}
static_assert(balanced_workers_per_cu(64) == 7 && balanced_workers_per_cu(96) == 5 &&
                  balanced_workers_per_cu(128) == 4,
              "workers per CU of the balanced schedule");

struct AcceptParams {
  const int32_t *proposals;    // [B][w]
  const int32_t *target_pred;  // [B][w]
  const int32_t *tested;       // [B] or null (= w)
  int32_t *accepted, *num_keep, *emitted, *num_emitted;  // emitted / num_emitted may be null
  uint32_t *dev_error;
  int32_t batch, w;
};
hipError_t launch_greedy_accept(const AcceptParams &p, hipStream_t s);

// Prefix split s of a sequence covers its pages [split_first_page(s),
// split_first_page(s + 1)); split 0 also carries the draft block (at most two
// 32-token tiles, one page's worth), so it holds one prefix page less and the
// splits of a sequence do equal work.
__host__ __device__ __forceinline__ int split_first_page(int s, int pps) {
  return s == 0 ? 0 : s * pps - 1;
}
// Splits of a sequence with `npages` prefix pages: ceil((npages + 1) / pps),
// at least 1 (the block's).
__host__ __device__ __forceinline__ int splits_of(int npages, int pps) {
  return (npages + pps) / pps;
}

// Launch geometry of the matrix-core kernel for a block of `rows` query rows
// (the launcher's template choice): 16-row tiles per wave and waves per
// workgroup.
__host__ __device__ constexpr int mfma_tiles_per_wave(int rows) { return rows <= 16 ? 1 : 2; }
__host__ __device__ constexpr int mfma_waves(int rows) {
  return rows <= 32 ? 1 : rows <= 64 ? 2 : 4;
}

// Query rows of one workgroup of the vector-ALU kernel: the smallest of 4, 8,
// 16 that holds the block's rows, else 32 (several row tiles).
__host__ __device__ constexpr int valu_tile_rows(int rows) {
  return rows <= 4 ? 4 : rows <= 8 ? 8 : rows <= 16 ? 16 : 32;
}

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------
typedef uint16_t bf16_t;  // raw bfloat16 bits

__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// Round to nearest, ties to even; NaN stays NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

__device__ __forceinline__ void report_error(uint32_t *word, uint32_t bits) {
  if (word) atomicOr(word, bits);
}

// Sequence prefix length, clamped to what the block table can address; an
// out-of-range value is reported once per sequence by the caller's thread 0.
__device__ __forceinline__ int clamp_prefix(int s, int max_pages, bool *bad) {
  const int cap = max_pages * kPage;
  *bad = (s < 0) || (s > cap);
  return s < 0 ? 0 : (s > cap ? cap : s);
}

}  // namespace das
