// Device building blocks shared by the matrix-core attention kernels:
// direct-to-LDS fragment loads, memory-counter waits, the bf16 MFMA, the
// 4-lane row reductions, and one 32-token tile through both products and
// the online softmax (Eq. (2)-(3)).
//
// MFMA 16x16x32 bf16 lane layout (lane l, n = l % 16, g = l / 16):
//   A[m][k]: lane holds m = n, k = 8g..8g+7   B[k][n]: k = 8g..8g+7, n
//   C[m][n]: lane holds m = 4g..4g+3, n
// Both products take the key / value tile as the A operand:
//   S^T (tokens x rows) = K_tile (tokens x dh) . Q^T (dh x rows)
//   O^T (dh x rows)    += V^T_tile (dh x tokens) . P^T (tokens x rows)
// so a lane's 8 probabilities of one query row (after exp2 and bf16
// rounding) are directly the B operand of the P.V product.
#pragma once

#include "das_internal.h"

namespace das {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kFragBytes = 64 * 16;  // one 16-byte fragment per lane

// 16 bytes per lane, global -> LDS at lds + 16 * lane (lds wave-uniform).
__device__ __forceinline__ void dma16(const void *src, uint8_t *lds) {
  __builtin_amdgcn_global_load_lds((__attribute__((address_space(1))) void *)(src),
                                   (__attribute__((address_space(3))) void *)(lds), 16, 0, 0);
}

// Raw buffer resource over `bytes` bytes at `base` (stride 0; word 3 = the
// gfx9 raw-buffer format). Out-of-range lanes read zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_of(const void *base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, 0x00020000);
}

// 16 bytes per lane from resource r at byte voff (per lane) + soff (uniform)
// -> LDS at lds + 16 * lane. The uniform part travels in an SGPR, so a
// fragment costs no vector address arithmetic. Cache policy: non-temporal
// (nt): prefix K/V are streamed once per call, and letting them displace the
// L2 like reused data cost 5-10 % of the rate on the batched workloads.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff,
                                      uint8_t *lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)(lds),
                                           16, voff, soff, 0, 2);
}

// s_waitcnt vmcnt(n), other counters untouched (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most `tiles` tiles of NF loads each are outstanding. Other
// loads or stores issued later only make the wait stricter.
template <int NF>
__device__ __forceinline__ void wait_tiles(int tiles) {
  if (tiles <= 0) wait_vmcnt<0>();
  else if (tiles == 1) wait_vmcnt<NF>();
  else if (tiles == 2) wait_vmcnt<(2 * NF < 64 ? 2 * NF : 0)>();
  else wait_vmcnt<(3 * NF < 64 ? 3 * NF : 0)>();
}

__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Reductions over the 4 lanes n, n + 16, n + 32, n + 48 (the rows of the C
// fragment that hold one query row): gfx950's permlane swaps exchange 16-lane
// rows (xor 16) and 32-lane halves (xor 32) between two registers in one
// VALU op, so with both operands = x the pair {x[l], x[l ^ 16]} (or
// {x[l], x[l ^ 32]}) lands in every lane; max and + are commutative, so the
// lanes of a group agree bit for bit.
__device__ __forceinline__ float group_max(float x) {
  const unsigned u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const unsigned v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group_sum(float x) {
  const unsigned u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const unsigned v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

typedef _Float16 h16x4 __attribute__((ext_vector_type(4)));

// One query row of a piece record (piece_record_bytes): the row's normalised
// output O / l in fp16, scaled by 2^-e so that its largest magnitude lies in
// [2^14, 2^15) (full fp16 precision for the row whatever the value scale,
// half the bytes of fp32 partials), and {m, l, q = l 2^e, 0}; the merge takes
// the row's unnormalised output as the stored values times q. m = -inf and
// l = 0 when no position was visible (weight 0 in the merge). Lane (n, g)
// holds head dims 16 dt + 4 g .. + 3 of the row; the 4 lanes of a row call
// this together (the row maximum is a 4-lane reduction).
template <int DH>
__device__ __forceinline__ void write_piece_row(uint8_t *rec, int rows, int row, int lg,
                                                const f32x4 (&o)[DH / 16], float m, float l) {
  const float inv = l > 0.f ? 1.f / l : 0.f;
  float amax = 0.f;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt)
#pragma unroll
    for (int v = 0; v < 4; ++v) amax = fmaxf(amax, fabsf(o[dt][v]));
  amax = group_max(amax) * inv;
  const int e = (amax > 0.f && amax < __builtin_huge_valf()) ? __builtin_amdgcn_frexp_expf(amax) - 15 : 0;
  const float sc = __builtin_amdgcn_ldexpf(inv, -e);
  _Float16 *orow = reinterpret_cast<_Float16 *>(rec) + row * DH;
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
    const h16x4 hv = {static_cast<_Float16>(o[dt][0] * sc), static_cast<_Float16>(o[dt][1] * sc),
                      static_cast<_Float16>(o[dt][2] * sc), static_cast<_Float16>(o[dt][3] * sc)};
    *reinterpret_cast<h16x4 *>(orow + 16 * dt + 4 * lg) = hv;
  }
  if (lg == 0) {
    const f32x4 meta = {m, l, __builtin_amdgcn_ldexpf(l, e), 0.f};
    *reinterpret_cast<f32x4 *>(rec + static_cast<size_t>(rows) * DH * 2 + row * 16) = meta;
  }
}

template <int DH, int NQ, int NB_>
struct Geo {
  static constexpr int KS = DH / 32;       // k steps of Q K^T
  static constexpr int DT = DH / 16;       // head-dim tiles of P V
  static constexpr int NF = 2 * KS + DT;   // fragments (loads) per 32-token tile
  static constexpr int SLOT = NF * kFragBytes;
  static constexpr int NB = NB_;           // ring depth
  static constexpr int QF = NQ * KS;       // Q fragments of a row tile
  static constexpr int LDS = NB * SLOT;
};

template <int DH, int NQ>
struct State {
  float m[NQ], l[NQ];
  f32x4 o[NQ][DH / 16];
};

// One 32-token tile through both products and the online softmax. Token t of
// the tile (0..31) is visible when t < limit and t <= cap[qt]; a full tile
// (every token visible) skips the mask.
// `hook(k)` runs between the stages (k = 0 before the logits, 1 before the
// softmax, 2 before P.V) so that the caller can spread work over the tile.
// LANE_SUM: st.l holds this lane's share of its row's sum (alpha is the same
// in a row's 4 lanes), which the caller reduces over the 4 lanes when it
// writes the row; otherwise st.l holds the row's sum after every tile.
template <int DH, int NQ, bool LANE_SUM = false, typename Hook>
__device__ __forceinline__ void compute_tile(State<DH, NQ> &st, const u32x4 (&kf)[2][DH / 32],
                                             const u32x4 (&vf)[DH / 16],
                                             const u32x4 (&qf)[NQ][DH / 32],
                                             const int (&cap)[NQ], int limit, bool full,
                                             float scale, int lg, Hook &&hook) {
  u16x8 pf[NQ];
  float alpha[NQ];
  bool moved[NQ];
  f32x4 sacc[NQ][2];
  hook(0);
  // k-step outermost: the 2 * NQ accumulators are independent, so no MFMA
  // waits for the one before it
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt)
#pragma unroll
    for (int e = 0; e < 2; ++e) sacc[qt][e] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < DH / 32; ++ks)
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt)
#pragma unroll
      for (int e = 0; e < 2; ++e) sacc[qt][e] = mfma16x16x32(kf[e][ks], qf[qt][ks], sacc[qt][e]);
  hook(1);
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    // raw logits; masked ones are -inf. scale > 0, so the maximum of the
    // scaled logits is the scaled maximum.
    float x[2][4];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int v = 0; v < 4; ++v) x[e][v] = sacc[qt][e][v];
    if (!full) {  // uniform: a full tile skips the mask
#pragma unroll
      for (int e = 0; e < 2; ++e) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int t = 8 * lg + 4 * e + v;
          x[e][v] = ((t < limit) & (t <= cap[qt])) ? x[e][v] : kNegInf;
        }
      }
    }
    float mx = kNegInf;
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int v = 0; v < 4; ++v) mx = fmaxf(mx, x[e][v]);
    // Running maximum (base-2 units): the row's largest probability is
    // exactly 1 and those near it fall just below, where bf16 rounds finest.
    mx = group_max(mx) * scale;
    const float mnew = fmaxf(st.m[qt], mx);
    const float neg = mnew == kNegInf ? 0.f : -mnew;  // nothing visible yet: every p is 0
    alpha[qt] = __builtin_amdgcn_exp2f(st.m[qt] + neg);
    moved[qt] = alpha[qt] != 1.f;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(x[e][v], scale, neg));
        psum += pv;
        pf[qt][4 * e + v] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(pv));
      }
    }
    if (!LANE_SUM) psum = group_sum(psum);
    st.l[qt] = st.l[qt] * alpha[qt] + psum;
    st.m[qt] = mnew;
  }
  hook(2);
  // rescale a row tile's accumulators only when the maximum of one of its
  // rows moved (a lane's accumulators of row tile qt all belong to one row)
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    if (__builtin_amdgcn_ballot_w64(moved[qt]) != 0) {
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) st.o[qt][dt] *= alpha[qt];
    }
  }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt)
      st.o[qt][dt] = mfma16x16x32(vf[dt], __builtin_bit_cast(u32x4, pf[qt]), st.o[qt][dt]);
  }
}

}  // namespace
}  // namespace das
