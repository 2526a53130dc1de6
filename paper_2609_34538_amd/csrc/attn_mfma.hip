// Matrix-core (MFMA) policy-attention kernel for bf16 caches (Eq. (2)-(3)).
//
// One workgroup = 4 waves on one (sequence, KV head, prefix split, row tile).
// The split's tiles are its 64-token prefix pages, plus the draft block on
// split 0; wave w takes tiles w, w+4, ... and keeps a private online-softmax
// state, with the next tile's key/value fragments loaded into registers while
// the current one is computed. The four states are merged through LDS.
// A sequence whose prefix fits one split is normalised and written out
// here; otherwise each split leaves its partial (O, m, l) in the workspace
// for the combine kernel.
//
// Both products run on v_mfma_f32_16x16x32_bf16 with the key/value tile as
// the A operand, so softmax probabilities never leave registers:
//   S^T (tokens x rows) = K_tile (tokens x dh) . Q^T (dh x rows)
//   O^T (dh x rows)    += V^T_tile (dh x tokens) . P^T (tokens x rows)
// MFMA 16x16x32 bf16 lane layout (lane l, n = l % 16, g = l / 16):
//   A[m][k]: lane holds m = n, k = 8g..8g+7   B[k][n]: k = 8g..8g+7, n
//   C[m][n]: lane holds m = 4g..4g+3, n
// The 16 token slots of each S^T tile are a permutation of the page tokens
// chosen so that the C fragments of tiles 2u and 2u+1 hold, per lane, the 8
// consecutive tokens 32u + 8g .. 32u + 8g + 7; those are exactly the k slots
// of the P^T fragment of the P.V product, and the matching V^T fragment is
// one contiguous 16-byte load from the dim-major value page.
//
// Query rows of a row tile: row = i * G + g (block position i, head
// kvh * G + g). Logits are scaled into base-2 units after the product.

#include "das_internal.h"

namespace das {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ u32x4 load16(const bf16_t *ptr) {
  return *reinterpret_cast<const u32x4 *>(ptr);
}

__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Token of the page/block held in slot m of S^T tile tt (see header comment).
__device__ __forceinline__ int slot_token(int tt, int m) {
  return 32 * (tt >> 1) + 8 * (m >> 2) + 4 * (tt & 1) + (m & 3);
}

// Key/value fragments of one half page (32 tokens, S^T tiles 2u and 2u+1).
template <int DH>
struct Frags {
  u32x4 k[2][DH / 32];
  u32x4 v[DH / 16];
};

template <int DH>
__device__ __forceinline__ void load_half(Frags<DH> &f, const bf16_t *kp, const bf16_t *vp,
                                          int u, int ln, int lg) {
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int tok = slot_token(2 * u + e, ln);
#pragma unroll
    for (int ks = 0; ks < DH / 32; ++ks) f.k[e][ks] = load16(kp + tok * DH + 32 * ks + 8 * lg);
  }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) f.v[dt] = load16(vp + (16 * dt + ln) * kPage + 32 * u + 8 * lg);
}

// Draft block half u: token-major K/V of stride Hkv * DH, w <= 64 tokens.
template <int DH>
__device__ __forceinline__ void load_block_half(Frags<DH> &f, const bf16_t *kb, const bf16_t *vb,
                                                int u, int w, size_t tok_stride, int ln, int lg) {
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int tok = slot_token(2 * u + e, ln);
#pragma unroll
    for (int ks = 0; ks < DH / 32; ++ks)
      f.k[e][ks] = tok < w ? load16(kb + tok * tok_stride + 32 * ks + 8 * lg) : u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    u16x8 v8;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int tok = 32 * u + 8 * lg + j;
      v8[j] = tok < w ? vb[tok * tok_stride + 16 * dt + ln] : static_cast<uint16_t>(0);
    }
    f.v[dt] = __builtin_bit_cast(u32x4, v8);
  }
}

template <int DH, int NQ>
struct State {
  float m[NQ], l[NQ];
  f32x4 o[NQ][DH / 16];
};

// One half page through both products and the online softmax. Token t of
// the half (0..31, page token 32u + t) is visible when t < limit for a
// prefix page, and when t < w - 32u and 32u + t <= i for the draft block.
template <int DH, int NQ>
__device__ __forceinline__ void compute_half(State<DH, NQ> &st, const Frags<DH> &f,
                                             const u32x4 (&qf)[NQ][DH / 32],
                                             const int (&row_i)[NQ], bool blk, int u, int limit,
                                             float scale, int lg) {
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    f32x4 sacc[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      sacc[e] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < DH / 32; ++ks) sacc[e] = mfma16x16x32(f.k[e][ks], qf[qt][ks], sacc[e]);
    }
    float x[2][4];
    float mx = kNegInf;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int t = 8 * lg + 4 * e + v;
        const bool vis = blk ? (t < limit && 32 * u + t <= row_i[qt]) : (t < limit);
        x[e][v] = vis ? sacc[e][v] * scale : kNegInf;
        mx = fmaxf(mx, x[e][v]);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mnew = fmaxf(st.m[qt], mx);
    const float muse = mnew == kNegInf ? 0.f : mnew;
    const float alpha = exp2f(st.m[qt] - muse);
    float psum = 0.f;
    u16x8 pf;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const __bf16 pb = static_cast<__bf16>(exp2f(x[e][v] - muse));
        psum += static_cast<float>(pb);
        pf[4 * e + v] = __builtin_bit_cast(uint16_t, pb);
      }
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    st.l[qt] = st.l[qt] * alpha + psum;
    st.m[qt] = mnew;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt)
      st.o[qt][dt] = mfma16x16x32(f.v[dt], __builtin_bit_cast(u32x4, pf), st.o[qt][dt] * alpha);
  }
}

template <int DH, int NQ>
__global__ __launch_bounds__(256) void attn_mfma_kernel(AttnParams p, int n_rt, int n_items) {
  constexpr int KS = DH / 32;
  constexpr int DT = DH / 16;
  constexpr int ROWS = 16 * NQ;
  constexpr int OS = DH + 1;    // padded LDS row stride of the merge buffer
  __shared__ float s_o[4][ROWS * OS];
  __shared__ float s_m[4][ROWS];
  __shared__ float s_l[4][ROWS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 15;
  const int lg = lane >> 4;

  // Workgroups are dealt to the 8 XCDs round-robin by linear id; the n_rt
  // row tiles of one (sequence, head, split) get ids 8 apart, so they run on
  // the same XCD and share its L2 for the key/value pages they all read.
  const int lin = blockIdx.x;
  const int rt = (lin >> 3) % n_rt;
  const int item = ((lin >> 3) / n_rt) * 8 + (lin & 7);
  if (item >= n_items) return;
  const int split = item % p.nsplit;
  const int unit = item / p.nsplit;
  const int kvh = unit % p.hkv;
  const int b = unit / p.hkv;
  const int pps = p.pages_per_split;
  const int pg0 = split * pps;

  // Independent loads first: prefix length, the page ids of this wave's
  // half-page tiles (wave w takes tiles w, w+4, ...; tile t is half t&1 of
  // page t>>1, so lane j holds the id of split page w/2 + 2j), and Q.
  const int s_raw = p.prefix_len[b];
  int my_page = 0;
  {
    const int pi = (wave >> 1) + 2 * lane;
    if (pi < pps && pg0 + pi < p.max_pages)
      my_page = p.block_table[static_cast<size_t>(b) * p.max_pages + pg0 + pi];
  }
  const int row_base = rt * ROWS;
  const bf16_t *q = static_cast<const bf16_t *>(p.q);
  u32x4 qf[NQ][KS];
  int row_i[NQ];
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    const int row = row_base + qt * 16 + ln;
    row_i[qt] = row / p.group;
    if (row < p.rows) {
      const int i = row / p.group, g = row % p.group;
      const bf16_t *qrow = q + ((static_cast<size_t>(b) * p.w + i) * p.hq + kvh * p.group + g) * DH;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[qt][ks] = load16(qrow + 32 * ks + 8 * lg);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[qt][ks] = u32x4{0, 0, 0, 0};
    }
  }

  bool bad_len;
  const int S = clamp_prefix(s_raw, p.max_pages, &bad_len);
  if (bad_len && split == 0 && kvh == 0 && rt == 0 && tid == 0)
    report_error(p.dev_error, DAS_DEVERR_PREFIX);
  const int npages = (S + kPage - 1) / kPage;
  const int n_pg = max(0, min(pps, npages - pg0));  // prefix pages of this split
  if (split > 0 && n_pg == 0) return;
  // half-page tiles: 2 per prefix page, then the block's halves on split 0
  const int ntiles = 2 * n_pg + (split == 0 ? (p.w + 31) / 32 : 0);
  int nsplit_b = (npages + pps - 1) / pps;
  if (nsplit_b < 1) nsplit_b = 1;

  const bf16_t *kl = static_cast<const bf16_t *>(p.k_layer);
  const bf16_t *vl = static_cast<const bf16_t *>(p.v_layer);
  const size_t head_off = static_cast<size_t>(kvh) * p.num_pages * kPage * DH;
  const bf16_t *kb = static_cast<const bf16_t *>(p.kb) +
                     (static_cast<size_t>(b) * p.w * p.hkv + kvh) * DH;
  const bf16_t *vb = static_cast<const bf16_t *>(p.vb) +
                     (static_cast<size_t>(b) * p.w * p.hkv + kvh) * DH;
  const size_t tok_stride = static_cast<size_t>(p.hkv) * DH;

  State<DH, NQ> st;
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    st.m[qt] = kNegInf;
    st.l[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) st.o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Tile t: half t&1 of prefix page t>>1 (t < 2 n_pg), else half
  // t - 2 n_pg of the block. Returns the visible-token limit of the half.
  auto issue = [&](Frags<DH> &f, int t) -> int {
    if (t < 2 * n_pg) {
      const int page = __builtin_amdgcn_readlane(my_page, (t - wave) >> 2);
      const bool ok = page >= 0 && page < p.num_pages;
      if (!ok && lane == 0) report_error(p.dev_error, DAS_DEVERR_PAGE);
      const size_t off = head_off + static_cast<size_t>(ok ? page : 0) * kPage * DH;
      load_half<DH>(f, kl + off, vl + off, t & 1, ln, lg);
      return ok ? min(32, S - (pg0 + (t >> 1)) * kPage - 32 * (t & 1)) : 0;
    }
    const int u = t - 2 * n_pg;
    load_block_half<DH>(f, kb, vb, u, p.w, tok_stride, ln, lg);
    return p.w - 32 * u;
  };

  Frags<DH> fa, fb;
  int t = wave;
  int lim_a = 0, lim_b = 0;
  if (t < ntiles) lim_a = issue(fa, t);
  while (t < ntiles) {
    if (t + 4 < ntiles) lim_b = issue(fb, t + 4);
    {
      const bool blk = t >= 2 * n_pg;
      compute_half<DH, NQ>(st, fa, qf, row_i, blk, blk ? t - 2 * n_pg : (t & 1), lim_a,
                           p.scale_log2, lg);
    }
    t += 4;
    if (t >= ntiles) break;
    if (t + 4 < ntiles) lim_a = issue(fa, t + 4);
    {
      const bool blk = t >= 2 * n_pg;
      compute_half<DH, NQ>(st, fb, qf, row_i, blk, blk ? t - 2 * n_pg : (t & 1), lim_b,
                           p.scale_log2, lg);
    }
    t += 4;
  }

  // Merge the four waves (each lane holds head dims 16dt+4g.. of row n).
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    const int r = qt * 16 + ln;
    if (lg == 0) {
      s_m[wave][r] = st.m[qt];
      s_l[wave][r] = st.l[qt];
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) s_o[wave][r * OS + 16 * dt + 4 * lg + v] = st.o[qt][dt][v];
    }
  }
  __syncthreads();

  bf16_t *out = static_cast<bf16_t *>(p.out);
  const int nrows = min(ROWS, p.rows - row_base);
  if (nsplit_b == 1) {
    // the whole prefix was this workgroup's: normalise and write the output
    for (int e = tid; e < nrows * DH; e += 256) {
      const int r = e / DH, c = e % DH;
      float mx = fmaxf(fmaxf(s_m[0][r], s_m[1][r]), fmaxf(s_m[2][r], s_m[3][r]));
      float o = 0.f, den = 0.f;
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) {
        const float sc = exp2f(s_m[w4][r] - mx);
        o += sc * s_o[w4][r * OS + c];
        den += sc * s_l[w4][r];
      }
      const int row = row_base + r;
      const int i = row / p.group, h = kvh * p.group + row % p.group;
      out[((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH + c] = f32_to_bf16(o / den);
      if (c == 0 && p.lse)
        p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] = (mx + log2f(den)) * 0.69314718055994530942f;
    }
    return;
  }

  // Partial of this split to the workspace.
  const size_t prow0 = ((static_cast<size_t>(b) * p.hkv + kvh) * p.nsplit + split) * p.rows + row_base;
  for (int e = tid; e < nrows * DH; e += 256) {
    const int r = e / DH, c = e % DH;
    float mx = fmaxf(fmaxf(s_m[0][r], s_m[1][r]), fmaxf(s_m[2][r], s_m[3][r]));
    if (mx == kNegInf) mx = 0.f;
    float o = 0.f, den = 0.f;
#pragma unroll
    for (int w4 = 0; w4 < 4; ++w4) {
      const float sc = exp2f(s_m[w4][r] - mx);
      o += sc * s_o[w4][r * OS + c];
      den += sc * s_l[w4][r];
    }
    p.ws_o[(prow0 + r) * DH + c] = o;
    if (c == 0) {
      p.ws_m[prow0 + r] = mx;
      p.ws_l[prow0 + r] = den;
    }
  }
}

template <int DH, int NQ>
hipError_t launch_typed(const AttnParams &p, hipStream_t s) {
  const int n_rt = (p.rows + 16 * NQ - 1) / (16 * NQ);
  const int n_items = p.batch * p.hkv * p.nsplit;
  const int grid = ((n_items + 7) / 8) * 8 * n_rt;
  hipLaunchKernelGGL((attn_mfma_kernel<DH, NQ>), dim3(grid), dim3(256), 0, s, p, n_rt, n_items);
  return hipGetLastError();
}

}  // namespace

int mfma_rows_per_wg(int rows) { return rows <= 16 ? 16 : 32; }

hipError_t launch_attn_mfma(const AttnParams &p, int dh, hipStream_t s) {
  const bool one = p.rows <= 16;
  if (dh == 64) return one ? launch_typed<64, 1>(p, s) : launch_typed<64, 2>(p, s);
  if (dh == 96) return one ? launch_typed<96, 1>(p, s) : launch_typed<96, 2>(p, s);
  return one ? launch_typed<128, 1>(p, s) : launch_typed<128, 2>(p, s);
}

}  // namespace das
