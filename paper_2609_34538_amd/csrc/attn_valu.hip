// Vector-ALU policy-attention kernel (Eq. (2)-(3)) over one prefix split.
//
// The only path for fp32 caches, and a bf16 path for comparison with the
// matrix-core kernel. One workgroup of four waves = (prefix split, KV head,
// sequence x row tile of RT query rows, RT = 4, 8, 16 or 32 chosen from the
// block's rows). The split's tiles (the draft block first on split 0, then
// its prefix pages) pass through LDS as fp32: keys token-major and values
// column-major, both in rows padded by 16 bytes so that 16 consecutive lanes
// reading 16 bytes each hit distinct banks. Wave v owns rows v, v + 4, ...;
// for the logits a lane is a token (its key row against broadcast query
// chunks), for P*V a lane is a head-dim column (its value column against
// broadcast probability chunks); every LDS read moves 16 bytes. The next
// tile's global loads are issued into registers before the current tile's
// arithmetic. Row max / sum are wave reductions over DPP and permlane swaps.
// The unnormalised partial (O, m, l) goes to the workspace and the combine
// kernel merges splits; a sequence that fits one split is written directly.

#include "das_internal.h"

namespace das {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

template <int CTRL> __device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}

// Butterfly over the 64 lanes: xor 1 and xor 2 inside a quad, the half-row
// mirror (lane i <-> 7 - i) and the row mirror (i <-> 15 - i) pair disjoint
// halves, then the permlane swaps cross 16-lane rows and 32-lane halves.
// Every step combines two disjoint lane sets with a commutative operation, so
// all lanes end with the same bits.
template <bool MAX> __device__ __forceinline__ float op(float a, float b) {
  return MAX ? fmaxf(a, b) : a + b;
}
template <bool MAX> __device__ __forceinline__ float wave_reduce(float x) {
  x = op<MAX>(x, dpp<0xB1>(x));
  x = op<MAX>(x, dpp<0x4E>(x));
  x = op<MAX>(x, dpp<0x141>(x));
  x = op<MAX>(x, dpp<0x140>(x));
  unsigned u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = op<MAX>(__uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(x);
  const auto c = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return op<MAX>(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

// Four consecutive cache elements as loaded (16 bytes of fp32, 8 of bf16).
template <typename T> struct Raw4;
template <> struct Raw4<float> {
  float4 v;
  __device__ __forceinline__ void load(const float *p) { v = *reinterpret_cast<const float4 *>(p); }
  __device__ __forceinline__ void zero() { v = make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ __forceinline__ float4 f() const { return v; }
};
template <> struct Raw4<bf16_t> {
  uint2 v;
  __device__ __forceinline__ void load(const bf16_t *p) { v = *reinterpret_cast<const uint2 *>(p); }
  __device__ __forceinline__ void zero() { v = make_uint2(0u, 0u); }
  __device__ __forceinline__ float4 f() const {
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
  }
};

__device__ __forceinline__ float4 lds4(const float *p) {
  return *reinterpret_cast<const float4 *>(p);
}
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float dot4(float4 a, float4 b, float s) {
  s = fmaf(a.x, b.x, s);
  s = fmaf(a.y, b.y, s);
  s = fmaf(a.z, b.z, s);
  return fmaf(a.w, b.w, s);
}

template <typename T, int DH, int RT>
__global__ __launch_bounds__(256) void attn_valu_kernel(AttnParams p) {
  constexpr int RW = RT / 4;          // rows per wave
  constexpr int KS = DH + 4;          // LDS row stride of the key tile (floats)
  constexpr int VS = kPage + 4;       // LDS row stride of the value tile (one column)
  constexpr int PS = kPage + 4;       // LDS row stride of the probabilities
  constexpr int NC = (DH + 63) / 64;  // head-dim columns per lane in P*V
  constexpr int NL = DH / 16;         // 4-element chunks of a tile per thread (K and V each)
  static_assert(DH % 16 == 0 && RT % 4 == 0, "tile shape");
  __shared__ __attribute__((aligned(16))) float sQ[RT * DH];
  __shared__ __attribute__((aligned(16))) float sK[kPage * KS];
  __shared__ __attribute__((aligned(16))) float sV[DH * VS];
  __shared__ __attribute__((aligned(16))) float sP[RT * PS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int n_rt = (p.rows + RT - 1) / RT;
  const int b = blockIdx.z / n_rt;
  const int rt = blockIdx.z % n_rt;

  const int row0 = rt * RT;
  const int nrows = min(RT, p.rows - row0);
  const int pg0 = split_first_page(split, p.pages_per_split);
  const int first_tile = (split == 0) ? -1 : pg0;  // -1 = the draft block
  const int32_t *table = p.block_table + static_cast<size_t>(b) * p.max_pages;
  // page id of a prefix tile (-1 past the table); its address does not
  // depend on the prefix length
  auto page_of = [&](int tile) { return tile >= 0 && tile < p.max_pages ? table[tile] : -1; };

  // One memory round trip before any arithmetic: the prefix length, the page
  // ids of the split's first two tiles and this row tile's Q are read
  // together, and the first tile's K/V follow its page id without waiting
  // for the prefix length. Every address stays in bounds whatever the length
  // turns out to be (a split past the prefix exits below).
  const int s_raw = p.prefix_len[b];
  int pid_cur = page_of(first_tile), pid_nxt = page_of(first_tile + 1);
  constexpr int QPT = (RT * DH + 255) / 256;  // Q elements per thread
  const T *q = static_cast<const T *>(p.q);
  float qv[QPT];
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = u * 256 + tid;
    const int r = e / DH, c = e % DH;
    qv[u] = 0.f;
    if (e < RT * DH && r < nrows) {
      const int row = row0 + r;
      const int i = row / p.group, g = row % p.group;
      const size_t off = ((static_cast<size_t>(b) * p.w + i) * p.hq + kvh * p.group + g) * DH + c;
      qv[u] = to_f32<T>(q[off]);
    }
  }

  const T *kl = static_cast<const T *>(p.k_layer);
  const T *vl = static_cast<const T *>(p.v_layer);
  const T *kb = static_cast<const T *>(p.kb);
  const T *vb = static_cast<const T *>(p.vb);
  const size_t head_elems = static_cast<size_t>(p.num_pages) * kPage * DH;

  // Thread tid's chunks of a tile are u * 256 + tid, u < NL: chunk e holds
  // elements 4e .. 4e + 3 of the key tile [64][DH] and of the value tile
  // ([8][DH][8] for a page, [w][Hkv][DH] rows for the draft block).
  Raw4<T> rk[NL], rv[NL];
  auto load_tile = [&](int tile, int page) {
    if (tile < 0) {
#pragma unroll
      for (int u = 0; u < NL; ++u) {
        const int e = u * 256 + tid;
        const int j = (4 * e) / DH, c = (4 * e) % DH;
        if (j < p.w) {
          const size_t off = ((static_cast<size_t>(b) * p.w + j) * p.hkv + kvh) * DH + c;
          rk[u].load(kb + off);
          rv[u].load(vb + off);
        } else {
          rk[u].zero();
          rv[u].zero();
        }
      }
    } else {
      // an unreadable page id reads page 0; its tokens are staged as zeros
      const bool ok = page >= 0 && page < p.num_pages;
      const size_t base = kvh * head_elems + static_cast<size_t>(ok ? page : 0) * kPage * DH;
#pragma unroll
      for (int u = 0; u < NL; ++u) {
        const int e = u * 256 + tid;
        rk[u].load(kl + base + 4 * e);
        rv[u].load(vl + base + 4 * e);
      }
    }
  };
  load_tile(first_tile, pid_cur);

  bool bad_len;
  const int S = clamp_prefix(s_raw, p.max_pages, &bad_len);
  if (bad_len && split == 0 && kvh == 0 && rt == 0 && tid == 0)
    report_error(p.dev_error, DAS_DEVERR_PREFIX);
  const int npages = (S + kPage - 1) / kPage;
  const int nsb = splits_of(npages, p.pages_per_split);  // this sequence's splits
  const int pg1 = min(split_first_page(split + 1, p.pages_per_split), npages);
  if (split > 0 && pg0 >= pg1) return;  // nothing to do; combine skips it

  // Q rows of this tile, pre-scaled into base-2 logit units.
#pragma unroll
  for (int u = 0; u < QPT; ++u) {
    const int e = u * 256 + tid;
    if (e < RT * DH) sQ[e] = qv[u] * p.scale_log2;
  }

  auto store_tile = [&](bool is_block, int valid) {
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const int e = u * 256 + tid;
      const int j = (4 * e) / DH, c = (4 * e) % DH;
      const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
      st4(&sK[j * KS + c], j < valid ? rk[u].f() : z);
      const float4 v = rv[u].f();
      if (is_block) {
        // rows [w][DH]: four columns of token j
        const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) sV[(c + t) * VS + j] = j < valid ? vv[t] : 0.f;
      } else {
        // page [8][DH][8]: tokens 8g + t0 .. + 3 of column cv
        const int g = (4 * e) / (8 * DH), cv = ((4 * e) % (8 * DH)) / 8, t0 = (4 * e) % 8;
        const int jv = 8 * g + t0;
        float4 w4;
        w4.x = jv < valid ? v.x : 0.f;
        w4.y = jv + 1 < valid ? v.y : 0.f;
        w4.z = jv + 2 < valid ? v.z : 0.f;
        w4.w = jv + 3 < valid ? v.w : 0.f;
        st4(&sV[cv * VS + jv], w4);
      }
    }
  };

  float m[RW], l[RW], acc[RW][NC];
#pragma unroll
  for (int k = 0; k < RW; ++k) {
    m[k] = kNegInf;
    l[k] = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[k][c] = 0.f;
  }

  for (int tile = first_tile; tile < pg1; ++tile) {
    const bool is_block = tile < 0;
    const bool ok = pid_cur >= 0 && pid_cur < p.num_pages;
    if (!is_block && !ok && tid == 0) report_error(p.dev_error, DAS_DEVERR_PAGE);
    // visible tokens of this tile: the block's w, a page's tokens before the
    // prefix length (none for an unreadable page); the rest are staged as zeros
    const int ntok = is_block ? p.w : (ok ? min(kPage, S - tile * kPage) : 0);
    __syncthreads();  // previous tile fully consumed (and sQ written)
    store_tile(is_block, ntok);
    __syncthreads();
    // the page id two tiles ahead and the next tile's K/V are in flight
    // during this tile
    const int pid_after = page_of(tile + 2);
    if (tile + 1 < pg1) load_tile(tile + 1, pid_nxt);
    pid_cur = pid_nxt;
    pid_nxt = pid_after;

    // Logits: lane = token j, this wave's RW rows.
    const int j = lane;
    float s[RW];
#pragma unroll
    for (int k = 0; k < RW; ++k) s[k] = 0.f;
#pragma unroll 2
    for (int i = 0; i < DH / 4; ++i) {
      const float4 kc = lds4(&sK[j * KS + 4 * i]);
#pragma unroll
      for (int k = 0; k < RW; ++k) s[k] = dot4(lds4(&sQ[(wave + 4 * k) * DH + 4 * i]), kc, s[k]);
    }
    float mt[RW];
#pragma unroll
    for (int k = 0; k < RW; ++k) {
      bool vis = j < ntok;
      if (is_block) vis = vis && j <= (row0 + wave + 4 * k) / p.group;
      s[k] = vis ? s[k] : kNegInf;
      mt[k] = wave_reduce<true>(s[k]);
    }
    float pj[RW], ps[RW];
#pragma unroll
    for (int k = 0; k < RW; ++k) {
      const float mn = fmaxf(m[k], mt[k]);
      const float mu = (mn == kNegInf) ? 0.f : mn;
      pj[k] = exp2f(s[k] - mu);
      const float alpha = exp2f(m[k] - mu);
      m[k] = mn;
      l[k] *= alpha;
#pragma unroll
      for (int c = 0; c < NC; ++c) acc[k][c] *= alpha;
      sP[(wave + 4 * k) * PS + j] = pj[k];
      ps[k] = wave_reduce<false>(pj[k]);
    }
#pragma unroll
    for (int k = 0; k < RW; ++k) l[k] += ps[k];
    __syncthreads();

    // P * V: lane = head-dim column(s), the wave's rows; tokens in fours up
    // to the last visible one (the rest have probability 0 and zero values).
    const int nq = (ntok + 3) / 4;
    for (int jq = 0; jq < nq; ++jq) {
      float4 pc[RW];
#pragma unroll
      for (int k = 0; k < RW; ++k) pc[k] = lds4(&sP[(wave + 4 * k) * PS + 4 * jq]);
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int col = lane + 64 * c;
        if (col < DH) {
          const float4 vc = lds4(&sV[col * VS + 4 * jq]);
#pragma unroll
          for (int k = 0; k < RW; ++k) acc[k][c] = dot4(pc[k], vc, acc[k][c]);
        }
      }
    }
  }

  // A sequence with a single split is normalised and written here (split 0
  // holds the block's diagonal, so l > 0); otherwise the unnormalised partial
  // of this split goes to the workspace for the combine kernel.
#pragma unroll
  for (int k = 0; k < RW; ++k) {
    const int r = wave + 4 * k;
    if (r >= nrows) continue;
    const int row = row0 + r;
    if (nsb == 1) {
      const float inv = 1.f / l[k];
      const int i = row / p.group, h = kvh * p.group + row % p.group;
      T *orow = static_cast<T *>(p.out) + ((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int col = lane + 64 * c;
        if (col < DH) orow[col] = from_f32<T>(acc[k][c] * inv);
      }
      if (lane == 0 && p.lse)
        p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] =
            (m[k] + log2f(l[k])) * 0.69314718055994530942f;
      continue;
    }
    const size_t prow = (((static_cast<size_t>(b) * p.hkv + kvh) * p.nsplit + split) * p.rows + row);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int col = lane + 64 * c;
      if (col < DH) p.ws_o[prow * DH + col] = acc[k][c];
    }
    if (lane == 0) {
      const size_t mrow =
          ((static_cast<size_t>(b) * p.hkv + kvh) * p.rows + row) * p.nsplit_ml + split;
      p.ws_m[mrow] = m[k];
      p.ws_l[mrow] = l[k];
    }
  }
}

template <typename T, int DH, int RT>
hipError_t launch_rt(const AttnParams &p, hipStream_t s) {
  const int n_rt = (p.rows + RT - 1) / RT;
  dim3 grid(p.nsplit, p.hkv, p.batch * n_rt);
  return launch_kernel(attn_valu_kernel<T, DH, RT>, grid, dim3(256), s, p);
}

template <typename T, int DH>
hipError_t launch_typed(const AttnParams &p, hipStream_t s) {
  switch (valu_tile_rows(p.rows)) {
    case 4: return launch_rt<T, DH, 4>(p, s);
    case 8: return launch_rt<T, DH, 8>(p, s);
    case 16: return launch_rt<T, DH, 16>(p, s);
    default: return launch_rt<T, DH, 32>(p, s);
  }
}

}  // namespace

hipError_t launch_attn_valu(const AttnParams &p, int dtype, int dh, hipStream_t s) {
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
