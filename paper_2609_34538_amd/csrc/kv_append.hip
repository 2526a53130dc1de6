// Commit of verified block K/V into the depth-indexed paged cache
// (Sec. 3.4: full-depth K/V of accepted, materialised inputs are retained;
// App. B.1: draft-side K/V never enter the cache).
//
// One wave per (plane, layer, KV head) of one sequence, four per workgroup,
// all of one sequence so the commit count n is uniform in the workgroup, and
// all keys or all values (the value waves share barriers).
// The wave reads the sequence's length, count and the (at most two) page ids
// its n new positions fall in once, then
//  - keys: copies the n token rows with 16-byte vectors (rows of head_dim
//    are contiguous in both the source and the token-major page);
//  - values: stages up to 16 token rows in LDS and writes them into the
//    token-grouped page ([8][dh][8]) transposed, lanes walking the token
//    index, so a wave's writes are runs of consecutive 16-byte groups.
// Pure copies: results are bit-exact.

#include "das_internal.h"

namespace das {
namespace {

constexpr int kWaves = 4;
constexpr int kChunk = 16;  // V tokens staged per pass

struct alignas(16) Vec16 {
  uint32_t x, y, z, w;
};

template <typename T, int DH>
__global__ __launch_bounds__(64 * kWaves) void kv_append_kernel(AppendParams p) {
  constexpr int VEC = 16 / sizeof(T);  // elements per 16-byte vector
  constexpr int NV = DH / VEC;         // vectors per token row
  __shared__ __attribute__((aligned(16))) T stage[kWaves][kChunk * DH];

  const int b = blockIdx.y;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int per_plane = p.layers * p.hkv;
  const int k_units = p.n_k_planes * per_plane, v_units = p.n_v_planes * per_plane;
  const int k_blocks = (k_units + kWaves - 1) / kWaves;
  const bool is_v = static_cast<int>(blockIdx.x) >= k_blocks;
  const int rel = (is_v ? blockIdx.x - k_blocks : blockIdx.x) * kWaves + wave;
  const bool live = rel < (is_v ? v_units : k_units);

  const int S = p.prefix_len[b];
  const int n = p.num_new[b];
  const bool bad = S < 0 || n < 0 || n > p.w_max ||
                   static_cast<long>(S) + n > static_cast<long>(p.max_pages) * kPage;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (bad) report_error(p.dev_error, DAS_DEVERR_COMMIT);
    if (p.len_out) p.len_out[b] = bad ? S : S + n;
  }
  if (bad || n == 0) return;  // uniform over the workgroup

  // n <= 64 new positions span at most two pages
  const int32_t *table = p.block_table + static_cast<size_t>(b) * p.max_pages;
  const int first_page = S / kPage;
  const int pg0 = table[first_page];
  const int pg1 = table[(S + n - 1) / kPage];
  const bool ok0 = pg0 >= 0 && pg0 < p.num_pages;
  const bool ok1 = pg1 >= 0 && pg1 < p.num_pages;
  if (blockIdx.x == 0 && threadIdx.x == 0 && (!ok0 || !ok1))
    report_error(p.dev_error, DAS_DEVERR_PAGE);

  const int plane = rel / per_plane;
  const int layer = (rel / p.hkv) % p.layers;
  const int h = rel % p.hkv;
  // source [plane][layer][B][w_max][Hkv][DH]; token t's row at src + t * hkv * DH
  const size_t src_off =
      ((((static_cast<size_t>(plane) * p.layers + layer) * p.batch + b) * p.w_max) * p.hkv + h) *
      DH;
  const size_t src_stride = static_cast<size_t>(p.hkv) * DH;
  // destination pages of this (plane, layer, head): [P][64 * DH]
  const size_t dst_head =
      ((static_cast<size_t>(plane) * p.layers + layer) * p.hkv + h) * p.num_pages * kPage * DH;

  if (!is_v) {
    if (!live) return;  // key workgroups use no barrier
    const T *src = static_cast<const T *>(p.k_new) + src_off;
    T *dst = static_cast<T *>(p.k_pool) + dst_head;
    const int total = n * NV;
    for (int v0 = 0; v0 < total; v0 += 4 * 64) {
      Vec16 r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < total) {
          const int t = v / NV, c = (v % NV) * VEC;
          r[u] = *reinterpret_cast<const Vec16 *>(src + t * src_stride + c);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = v0 + u * 64 + lane;
        if (v < total) {
          const int t = v / NV, c = (v % NV) * VEC;
          const int pos = S + t;
          const bool second = pos / kPage != first_page;
          if (second ? ok1 : ok0) {
            const size_t page = second ? pg1 : pg0;
            *reinterpret_cast<Vec16 *>(dst + (page * kPage + pos % kPage) * DH + c) = r[u];
          }
        }
      }
    }
    return;
  }

  // values: every wave of the workgroup, live or not, runs the same chunk
  // loop and its barriers (n is uniform)
  const T *src = static_cast<const T *>(p.v_new) + src_off;
  T *dst = static_cast<T *>(p.v_pool) + dst_head;
  T *st = stage[wave];
  for (int t0 = 0; t0 < n; t0 += kChunk) {
    const int tc = min(kChunk, n - t0);
    if (live) {
      for (int v = lane; v < tc * NV; v += 64) {
        const int t = v / NV, c = (v % NV) * VEC;
        *reinterpret_cast<Vec16 *>(st + t * DH + c) =
            *reinterpret_cast<const Vec16 *>(src + (t0 + t) * src_stride + c);
      }
    }
    __syncthreads();
    if (live) {
      for (int e = lane; e < tc * DH; e += 64) {
        const int c = e / tc, t = e % tc;
        const int pos = S + t0 + t;
        const bool second = pos / kPage != first_page;
        if (second ? ok1 : ok0) {
          const size_t page = second ? pg1 : pg0;
          dst[page * kPage * DH + ((pos % kPage) / 8 * DH + c) * 8 + pos % 8] = st[t * DH + c];
        }
      }
    }
    __syncthreads();
  }
}

template <typename T, int DH>
hipError_t launch_typed(const AppendParams &p, hipStream_t s) {
  const int per_plane = p.layers * p.hkv;
  const int blocks = (p.n_k_planes * per_plane + kWaves - 1) / kWaves +
                     (p.n_v_planes * per_plane + kWaves - 1) / kWaves;
  dim3 grid(blocks, p.batch);
  hipLaunchKernelGGL((kv_append_kernel<T, DH>), grid, dim3(64 * kWaves), 0, s, p);
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
