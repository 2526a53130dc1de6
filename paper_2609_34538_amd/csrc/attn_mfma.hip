// Matrix-core (MFMA) policy-attention kernel for bf16 caches (Eq. (2)-(3)).
//
// One workgroup = 4 waves on one (sequence, KV head, prefix split, row tile).
// The waves take the split's tiles round-robin (the draft block first on
// split 0, then 64-token prefix pages) and keep private online-softmax
// states, merged through LDS at the end into one partial (O, m, l) per split.
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

// Token of page/block held in slot m of S^T tile tt (see header comment).
__device__ __forceinline__ int slot_token(int tt, int m) {
  return 32 * (tt >> 1) + 8 * (m >> 2) + 4 * (tt & 1) + (m & 3);
}

template <int DH, int NQ>
__global__ __launch_bounds__(256) void attn_mfma_kernel(AttnParams p, int n_rt, int n_items) {
  constexpr int KS = DH / 32;   // k steps of the Q K^T product
  constexpr int DT = DH / 16;   // head-dim tiles of the P V product
  constexpr int ROWS = 16 * NQ;
  constexpr int OS = DH + 1;    // padded LDS row stride of the merge buffer
  __shared__ float s_o[4][ROWS * OS];
  __shared__ float s_m[4][ROWS];
  __shared__ float s_l[4][ROWS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
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

  bool bad_len;
  const int S = clamp_prefix(p.prefix_len[b], p.max_pages, &bad_len);
  if (bad_len && split == 0 && kvh == 0 && rt == 0 && tid == 0)
    report_error(p.dev_error, DAS_DEVERR_PREFIX);
  const int npages = (S + kPage - 1) / kPage;
  const int pg0 = split * p.pages_per_split;
  const int pg1 = min(pg0 + p.pages_per_split, npages);
  if (split > 0 && pg0 >= pg1) return;

  const int row_base = rt * ROWS;
  const bf16_t *q = static_cast<const bf16_t *>(p.q);
  const bf16_t *kb = static_cast<const bf16_t *>(p.kb);
  const bf16_t *vb = static_cast<const bf16_t *>(p.vb);
  const bf16_t *kl = static_cast<const bf16_t *>(p.k_layer);
  const bf16_t *vl = static_cast<const bf16_t *>(p.v_layer);

  // Q^T fragments (B operand): row n of each 16-row tile, head dims 32ks+8g..
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

  float m_run[NQ], l_run[NQ];
  f32x4 oacc[NQ][DT];
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    m_run[qt] = kNegInf;
    l_run[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int has_block = split == 0 ? 1 : 0;
  const int ntiles = has_block + max(0, pg1 - pg0);
  const size_t head_elems = static_cast<size_t>(p.num_pages) * kPage * DH;

  for (int ti = wave; ti < ntiles; ti += 4) {
    const bool blk = has_block && ti == 0;
    const int tile = blk ? -1 : pg0 + ti - has_block;
    u32x4 kf[4][KS];
    u32x4 vf[DT][2];
    bool ok = true;
    if (blk) {
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const int tok = slot_token(tt, ln);
        const bf16_t *krow = kb + ((static_cast<size_t>(b) * p.w + tok) * p.hkv + kvh) * DH;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          kf[tt][ks] = tok < p.w ? load16(krow + 32 * ks + 8 * lg) : u32x4{0, 0, 0, 0};
      }
      // block values are token-major: gather 8 tokens per fragment
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          u16x8 v8;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int tok = 32 * u + 8 * lg + j;
            v8[j] = tok < p.w
                        ? vb[((static_cast<size_t>(b) * p.w + tok) * p.hkv + kvh) * DH + 16 * dt + ln]
                        : static_cast<uint16_t>(0);
          }
          vf[dt][u] = __builtin_bit_cast(u32x4, v8);
        }
      }
    } else {
      const int page = p.block_table[static_cast<size_t>(b) * p.max_pages + tile];
      ok = page >= 0 && page < p.num_pages;
      if (!ok && lane == 0) report_error(p.dev_error, DAS_DEVERR_PAGE);
      const size_t base = kvh * head_elems + static_cast<size_t>(ok ? page : 0) * kPage * DH;
      const bf16_t *kp = kl + base;   // [64][DH]
      const bf16_t *vp = vl + base;   // [DH][64]
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const int tok = slot_token(tt, ln);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[tt][ks] = load16(kp + tok * DH + 32 * ks + 8 * lg);
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int u = 0; u < 2; ++u) vf[dt][u] = load16(vp + (16 * dt + ln) * kPage + 32 * u + 8 * lg);
      }
    }

#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      f32x4 sacc[4];
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        sacc[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sacc[tt] = mfma16x16x32(kf[tt][ks], qf[qt][ks], sacc[tt]);
      }
      // mask, scale, online softmax over this tile (row n = ln of tile qt)
      float x[4][4];
      float mx = kNegInf;
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int tok = 32 * (tt >> 1) + 8 * lg + 4 * (tt & 1) + v;
          const bool vis = blk ? (tok < p.w && tok <= row_i[qt])
                               : (ok && tile * kPage + tok < S);
          x[tt][v] = vis ? sacc[tt][v] * p.scale_log2 : kNegInf;
          mx = fmaxf(mx, x[tt][v]);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(m_run[qt], mx);
      const float muse = mnew == kNegInf ? 0.f : mnew;
      const float alpha = exp2f(m_run[qt] - muse);
      float psum = 0.f;
      u16x8 pf[2];
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const __bf16 pb = static_cast<__bf16>(exp2f(x[tt][v] - muse));
          psum += static_cast<float>(pb);
          pf[tt >> 1][4 * (tt & 1) + v] = __builtin_bit_cast(uint16_t, pb);
        }
      }
      psum += __shfl_xor(psum, 16, 64);
      psum += __shfl_xor(psum, 32, 64);
      l_run[qt] = l_run[qt] * alpha + psum;
      m_run[qt] = mnew;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        oacc[qt][dt] *= alpha;
#pragma unroll
        for (int u = 0; u < 2; ++u)
          oacc[qt][dt] = mfma16x16x32(vf[dt][u], __builtin_bit_cast(u32x4, pf[u]), oacc[qt][dt]);
      }
    }
  }

  // Merge the four waves' states (each lane holds head dims 16dt+4g.. of row n).
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    const int r = qt * 16 + ln;
    if (lg == 0) {
      s_m[wave][r] = m_run[qt];
      s_l[wave][r] = l_run[qt];
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) s_o[wave][r * OS + 16 * dt + 4 * lg + v] = oacc[qt][dt][v];
    }
  }
  __syncthreads();
  const size_t prow0 = ((static_cast<size_t>(b) * p.hkv + kvh) * p.nsplit + split) * p.rows;
  for (int e = tid; e < ROWS * DH; e += 256) {
    const int r = e / DH, c = e % DH;
    const int row = row_base + r;
    if (row >= p.rows) continue;
    float mx = fmaxf(fmaxf(s_m[0][r], s_m[1][r]), fmaxf(s_m[2][r], s_m[3][r]));
    if (mx == kNegInf) mx = 0.f;
    float o = 0.f, den = 0.f;
#pragma unroll
    for (int w4 = 0; w4 < 4; ++w4) {
      const float sc = exp2f(s_m[w4][r] - mx);
      o += sc * s_o[w4][r * OS + c];
      den += sc * s_l[w4][r];
    }
    p.ws_o[(prow0 + row) * DH + c] = o;
    if (c == 0) {
      p.ws_m[prow0 + row] = mx;
      p.ws_l[prow0 + row] = den;
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
