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
//  - values: stages up to 16 token rows in LDS; then each lane takes one
//    (head dim, 8-position group) of the token-grouped page ([8][dh][8]),
//    whose new positions are one contiguous run, and writes the run with
//    the widest aligned stores that fit it (a full group is one 16-byte
//    store for bf16).
// Pure copies: results are bit-exact.

#include "das_internal.h"

namespace das {
namespace {

constexpr int kWaves = 4;
constexpr int kChunk = 16;  // V tokens staged per pass

struct alignas(16) Vec16 {
  uint32_t x, y, z, w;
};

// 32-bit words of elements (two bf16 per word, one fp32 per word).
__device__ __forceinline__ uint32_t word(const bf16_t (&v)[8], int i) {
  return static_cast<uint32_t>(v[2 * i]) | (static_cast<uint32_t>(v[2 * i + 1]) << 16);
}
__device__ __forceinline__ uint32_t word(const float (&v)[8], int i) {
  return __float_as_uint(v[i]);
}

// Elements [lo, hi) of an 8-element row (16-byte aligned for bf16, 32 for
// fp32) from v[], in aligned pieces of at most 16 bytes. Every piece position
// is a compile-time constant, so v[] stays in registers.
template <typename T>
__device__ __forceinline__ void store_run(T *row, const T (&v)[8], int lo, int hi) {
  constexpr int EPW = 4 / sizeof(T);  // elements per 32-bit word
  auto inside = [&](int a, int b) { return lo <= a && b <= hi; };
  if constexpr (sizeof(T) == 2) {
    if (inside(0, 8)) {
      *reinterpret_cast<Vec16 *>(row) = Vec16{word(v, 0), word(v, 1), word(v, 2), word(v, 3)};
      return;
    }
  }
#pragma unroll
  for (int q = 0; q < 8; q += 4) {
    if (inside(q, q + 4)) {  // 8 bytes (bf16) or 16 bytes (fp32)
      const int w0 = q / EPW;
      if constexpr (sizeof(T) == 2) {
        *reinterpret_cast<uint2 *>(row + q) = make_uint2(word(v, w0), word(v, w0 + 1));
      } else {
        *reinterpret_cast<Vec16 *>(row + q) =
            Vec16{word(v, w0), word(v, w0 + 1), word(v, w0 + 2), word(v, w0 + 3)};
      }
      continue;
    }
#pragma unroll
    for (int e = q; e < q + 4; e += 2) {
      if (inside(e, e + 2)) {  // 4 bytes (bf16) or 8 bytes (fp32)
        if constexpr (sizeof(T) == 2) {
          *reinterpret_cast<uint32_t *>(row + e) = word(v, e / 2);
        } else {
          *reinterpret_cast<uint2 *>(row + e) = make_uint2(word(v, e), word(v, e + 1));
        }
        continue;
      }
      if (inside(e, e + 1)) row[e] = v[e];
      if (inside(e + 1, e + 2)) row[e + 1] = v[e + 1];
    }
  }
}

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
    // vector v: token v / NV, columns (v % NV) * VEC ..
    auto load = [&](int v) {
      Vec16 r = {0, 0, 0, 0};
      if (v < total) r = *reinterpret_cast<const Vec16 *>(src + (v / NV) * src_stride + (v % NV) * VEC);
      return r;
    };
    auto store = [&](int v, const Vec16 &r) {
      if (v >= total) return;
      const int t = v / NV, c = (v % NV) * VEC;
      const int pos = S + t;
      const bool second = pos / kPage != first_page;
      if (second ? ok1 : ok0) {
        const size_t page = second ? pg1 : pg0;
        *reinterpret_cast<Vec16 *>(dst + (page * kPage + pos % kPage) * DH + c) = r;
      }
    };
    for (int v0 = lane; v0 < total; v0 += 4 * 64) {
      const Vec16 r0 = load(v0), r1 = load(v0 + 64), r2 = load(v0 + 128), r3 = load(v0 + 192);
      store(v0, r0);
      store(v0 + 64, r1);
      store(v0 + 128, r2);
      store(v0 + 192, r3);
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
      // item (dim c, 8-position group gi): the chunk's positions in that group
      // are one contiguous run of the page's [group][c][8] row, written with
      // the widest aligned stores that fit it
      const int p0 = S + t0, p1 = p0 + tc;
      const int gbase = p0 & ~7;
      const int ngroups = (p1 - gbase + 7) >> 3;
      for (int item = lane; item < DH * ngroups; item += 64) {
        const int c = item % DH, gp = gbase + 8 * (item / DH);
        const int lo = max(gp, p0), hi = min(gp + 8, p1);
        const bool second = gp / kPage != first_page;  // 8 | 64: a group lies in one page
        if (!(second ? ok1 : ok0)) continue;
        const size_t page = second ? pg1 : pg0;
        T *row = dst + page * kPage * DH + ((gp % kPage) / 8 * DH + c) * 8;
        T v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int t = min(max(gp + j - p0, 0), tc - 1);  // staged token index
          v[j] = (gp + j >= lo && gp + j < hi) ? st[t * DH + c] : T(0);
        }
        store_run<T>(row, v, lo - gp, hi - gp);
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
  return launch_kernel(kv_append_kernel<T, DH>, grid, dim3(64 * kWaves), s, p);
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
