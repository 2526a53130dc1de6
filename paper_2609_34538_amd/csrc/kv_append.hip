// Commit of verified block K/V into the depth-indexed paged cache
// (Sec. 3.4: full-depth K/V of accepted, materialised inputs are retained;
// App. B.1: draft-side K/V never enter the cache).
//
// One workgroup per (sequence, plane x layer x KV head). Keys are copied
// token by token (rows of head_dim contiguous in both source and page);
// values are written into dim-major pages, so lanes walk the token index to
// keep the page writes contiguous. Pure copies: results are bit-exact.

#include "das_internal.h"

namespace das {
namespace {

template <typename T, int DH>
__global__ __launch_bounds__(256) void kv_append_kernel(AppendParams p) {
  const int b = blockIdx.x;
  const int sel = blockIdx.y;  // (plane, layer, head) over K planes then V planes
  const int per_plane = p.layers * p.hkv;
  const bool is_v = sel >= p.n_k_planes * per_plane;
  const int rel = is_v ? sel - p.n_k_planes * per_plane : sel;
  const int plane = rel / per_plane;
  const int layer = (rel / p.hkv) % p.layers;
  const int h = rel % p.hkv;

  const int s_raw = p.prefix_len[b];
  const int n_raw = p.num_new[b];
  const bool bad = s_raw < 0 || n_raw < 0 || n_raw > p.w_max ||
                   static_cast<long>(s_raw) + n_raw > static_cast<long>(p.max_pages) * kPage;
  if (sel == 0 && threadIdx.x == 0) {
    if (bad) report_error(p.dev_error, DAS_DEVERR_COMMIT);
    if (p.len_out) p.len_out[b] = bad ? s_raw : s_raw + n_raw;
  }
  if (bad || n_raw == 0) return;
  const int S = s_raw, n = n_raw;

  // source [plane][layer][B][w_max][Hkv][DH]
  const size_t src_base =
      (((static_cast<size_t>(plane) * p.layers + layer) * p.batch + b) * p.w_max) * p.hkv * DH;
  // destination [plane][layer][Hkv][P] pages of 64 * DH elements
  const size_t dst_head =
      ((static_cast<size_t>(plane) * p.layers + layer) * p.hkv + h) * p.num_pages * kPage * DH;
  const int32_t *table = p.block_table + static_cast<size_t>(b) * p.max_pages;

  if (!is_v) {
    const T *src = static_cast<const T *>(p.k_new);
    T *dst = static_cast<T *>(p.k_pool);
    for (int e = threadIdx.x; e < n * DH; e += blockDim.x) {
      const int t = e / DH, c = e % DH;
      const int pos = S + t;
      const int page = table[pos / kPage];
      if (page < 0 || page >= p.num_pages) {
        report_error(p.dev_error, DAS_DEVERR_PAGE);
        continue;
      }
      dst[dst_head + (static_cast<size_t>(page) * kPage + pos % kPage) * DH + c] =
          src[src_base + (static_cast<size_t>(t) * p.hkv + h) * DH + c];
    }
  } else {
    const T *src = static_cast<const T *>(p.v_new);
    T *dst = static_cast<T *>(p.v_pool);
    for (int e = threadIdx.x; e < n * DH; e += blockDim.x) {
      const int c = e / n, t = e % n;
      const int pos = S + t;
      const int page = table[pos / kPage];
      if (page < 0 || page >= p.num_pages) {
        report_error(p.dev_error, DAS_DEVERR_PAGE);
        continue;
      }
      dst[dst_head + (static_cast<size_t>(page) * DH + c) * kPage + pos % kPage] =
          src[src_base + (static_cast<size_t>(t) * p.hkv + h) * DH + c];
    }
  }
}

template <typename T, int DH>
hipError_t launch_typed(const AppendParams &p, hipStream_t s) {
  dim3 grid(p.batch, (p.n_k_planes + p.n_v_planes) * p.layers * p.hkv);
  hipLaunchKernelGGL((kv_append_kernel<T, DH>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_kv_append(const AppendParams &p, int dtype, int dh, hipStream_t s) {
  if (dtype == DAS_F32) {
    if (dh == 64) return launch_typed<float, 64>(p, s);
    if (dh == 96) return launch_typed<float, 96>(p, s);
    return launch_typed<float, 128>(p, s);
  }
  if (dh == 64) return launch_typed<bf16_t, 64>(p, s);
  if (dh == 96) return launch_typed<bf16_t, 96>(p, s);
  return launch_typed<bf16_t, 128>(p, s);
}

}  // namespace das
