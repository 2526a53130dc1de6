// Vector-ALU policy-attention kernel (Eq. (2)-(3)) over one prefix split.
//
// The only path for fp32 caches, and a bf16 path for comparison with the
// matrix-core kernel. One workgroup = (prefix split, KV head, sequence x row
// tile of up to 32 query rows). The split's tiles (the draft block first on
// split 0, then its prefix pages) are staged through LDS as fp32; each wave
// owns 8 query rows, lanes map to tokens for the logits and to head-dim
// columns for P*V, and the online-softmax row max / sum are wave reductions.
// The unnormalised partial (O, m, l) goes to the workspace; the combine
// kernel merges splits.

#include "das_internal.h"

namespace das {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_valu_kernel(AttnParams p) {
  constexpr int RT = kValuRows;        // rows per workgroup
  constexpr int RW = RT / 4;           // rows per wave
  constexpr int KS = DH + 1;           // padded LDS row stride of the key tile
  constexpr int VS = kPage + 1;        // padded LDS row stride of the value tile
  constexpr int NC = (DH + 63) / 64;   // head-dim columns per lane
  __shared__ float sQ[RT * DH];
  __shared__ float sK[kPage * KS];
  __shared__ float sV[DH * VS];
  __shared__ float sP[RT * (kPage + 1)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int n_rt = (p.rows + RT - 1) / RT;
  const int b = blockIdx.z / n_rt;
  const int rt = blockIdx.z % n_rt;

  bool bad_len;
  const int S = clamp_prefix(p.prefix_len[b], p.max_pages, &bad_len);
  if (bad_len && split == 0 && kvh == 0 && rt == 0 && tid == 0)
    report_error(p.dev_error, DAS_DEVERR_PREFIX);
  const int npages = (S + kPage - 1) / kPage;
  const int pg0 = split_first_page(split, p.pages_per_split);
  const int pg1 = min(split_first_page(split + 1, p.pages_per_split), npages);
  if (split > 0 && pg0 >= pg1) return;  // nothing to do; combine skips it

  const int row0 = rt * RT;
  const int nrows = min(RT, p.rows - row0);
  const T *q = static_cast<const T *>(p.q);
  // Q rows of this tile, pre-scaled into base-2 logit units.
  for (int e = tid; e < RT * DH; e += 256) {
    const int r = e / DH, c = e % DH;
    float v = 0.f;
    if (r < nrows) {
      const int row = row0 + r;
      const int i = row / p.group, g = row % p.group;
      const size_t off = ((static_cast<size_t>(b) * p.w + i) * p.hq + kvh * p.group + g) * DH + c;
      v = to_f32<T>(q[off]) * p.scale_log2;
    }
    sQ[e] = v;
  }

  float m[RW], l[RW], acc[RW][NC];
#pragma unroll
  for (int k = 0; k < RW; ++k) {
    m[k] = kNegInf;
    l[k] = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[k][c] = 0.f;
  }

  const T *kl = static_cast<const T *>(p.k_layer);
  const T *vl = static_cast<const T *>(p.v_layer);
  const size_t head_elems = static_cast<size_t>(p.num_pages) * kPage * DH;
  const int first_tile = (split == 0) ? -1 : pg0;  // -1 = the draft block

  for (int tile = first_tile; tile < pg1; ++tile) {
    const bool is_block = tile < 0;
    int ntok = kPage;
    __syncthreads();  // previous tile fully consumed
    if (is_block) {
      ntok = p.w;
      const T *kb = static_cast<const T *>(p.kb);
      const T *vb = static_cast<const T *>(p.vb);
      for (int e = tid; e < kPage * DH; e += 256) {
        const int j = e / DH, c = e % DH;
        float kv = 0.f, vv = 0.f;
        if (j < ntok) {
          const size_t off = ((static_cast<size_t>(b) * p.w + j) * p.hkv + kvh) * DH + c;
          kv = to_f32<T>(kb[off]);
          vv = to_f32<T>(vb[off]);
        }
        sK[j * KS + c] = kv;
        sV[c * VS + j] = vv;
      }
    } else {
      int page = p.block_table[static_cast<size_t>(b) * p.max_pages + tile];
      bool ok = page >= 0 && page < p.num_pages;
      if (!ok && tid == 0) report_error(p.dev_error, DAS_DEVERR_PAGE);
      const size_t base = kvh * head_elems + static_cast<size_t>(ok ? page : 0) * kPage * DH;
      // tokens past the prefix (and an unreadable page) are staged as zeros:
      // they enter P.V with probability 0, whatever the cache holds there
      const int valid = ok ? min(kPage, S - tile * kPage) : 0;
      for (int e = tid; e < kPage * DH; e += 256) {
        // key tile is [64][DH], value tile is [8][DH][8]; both contiguous
        const int j = e / DH, c = e % DH;
        sK[j * KS + c] = j < valid ? to_f32<T>(kl[base + e]) : 0.f;
        const int cv = (e >> 3) % DH, jv = 8 * (e / (8 * DH)) + (e & 7);
        sV[cv * VS + jv] = jv < valid ? to_f32<T>(vl[base + e]) : 0.f;
      }
      if (!ok) ntok = 0;  // skip the unreadable page
    }
    __syncthreads();

    // Logits: lane = token, this wave's RW rows.
    const int j = lane;
    const int pos = is_block ? j : tile * kPage + j;
#pragma unroll
    for (int k = 0; k < RW; ++k) {
      const int r = wave + 4 * k;
      float s = 0.f;
#pragma unroll 8
      for (int c = 0; c < DH; ++c) s += sQ[r * DH + c] * sK[j * KS + c];
      bool vis;
      if (is_block) {
        const int i = (row0 + r) / p.group;
        vis = (j < ntok) && (j <= i);
      } else {
        vis = (j < ntok) && (pos < S);
      }
      s = vis ? s : kNegInf;
      const float mt = wave_max(s);
      const float mn = fmaxf(m[k], mt);
      const float mu = (mn == kNegInf) ? 0.f : mn;
      const float pj = exp2f(s - mu);
      const float alpha = exp2f(m[k] - mu);
      l[k] = l[k] * alpha + wave_sum(pj);
      m[k] = mn;
#pragma unroll
      for (int c = 0; c < NC; ++c) acc[k][c] *= alpha;
      sP[r * (kPage + 1) + j] = pj;
    }
    __syncthreads();

    // P * V: lane = head-dim column(s), the wave's rows.
    for (int jj = 0; jj < ntok; ++jj) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int col = lane + 64 * c;
        if (col < DH) {
          const float v = sV[col * VS + jj];
#pragma unroll
          for (int k = 0; k < RW; ++k) acc[k][c] += sP[(wave + 4 * k) * (kPage + 1) + jj] * v;
        }
      }
    }
  }

  // Unnormalised partial results of this split.
#pragma unroll
  for (int k = 0; k < RW; ++k) {
    const int r = wave + 4 * k;
    if (r >= nrows) continue;
    const int row = row0 + r;
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

template <typename T, int DH>
hipError_t launch_typed(const AttnParams &p, hipStream_t s) {
  const int n_rt = (p.rows + kValuRows - 1) / kValuRows;
  dim3 grid(p.nsplit, p.hkv, p.batch * n_rt);
  hipLaunchKernelGGL((attn_valu_kernel<T, DH>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
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
