// Merge of the per-split partial results into the attention output.
//
// Each split s of a (sequence, KV head) left, per query row, an unnormalised
// output O_s, its running maximum m_s (base-2 logit units) and its running
// sum l_s. With M = max_s m_s the joint softmax of Eq. (2) over all splits is
//   O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,
// and the natural-log normaliser is (M + log2 sum_s 2^(m_s - M) l_s) * ln 2.
// Split 0 always holds the block's diagonal, so M is finite.

#include "mfma_tile.h"

namespace das {
namespace {

constexpr int kRowsPerBlock = 8;
constexpr int kColsPerBlock = 32;
constexpr int kEager = 24;  // splits whose partials are loaded before the count is known

// One single-wave workgroup per (sequence, KV head, 8 rows, 32 columns); one
// thread per (row, 4 consecutive columns). A row's per-split maxima and sums
// are contiguous, so they arrive as 16-byte vectors; the partials of the first
// 24 splits the workspace holds are loaded together with the prefix length,
// so a merge of up to 24 splits costs one memory round trip. Values of splits
// past the sequence's count are discarded by selection, never used in
// arithmetic.
template <typename T, int DH>
__global__ __launch_bounds__(64) void attn_combine_kernel(AttnParams p, int skip_single) {
  const int unit = blockIdx.x;  // b * hkv + kvh
  const int b = unit / p.hkv;
  const int kvh = unit % p.hkv;
  const int row = blockIdx.y * kRowsPerBlock + threadIdx.x / 8;
  const int c = blockIdx.z * kColsPerBlock + 4 * (threadIdx.x % 8);
  const bool live = row < p.rows && c < DH;
  const int r0 = live ? row : 0, c0 = live ? c : 0;
  const size_t obase = (static_cast<size_t>(unit) * p.nsplit) * p.rows + r0;  // split 0's row
  const size_t mbase = (static_cast<size_t>(unit) * p.rows + r0) * p.nsplit_ml;

  const int s_raw = p.prefix_len[b];
  float mv[kEager], lv[kEager];
  float4 ov[kEager];
#pragma unroll
  for (int k4 = 0; k4 < kEager / 4; ++k4) {
    // the row's nsplit_ml (a multiple of 4) slots; split slots past the
    // plan's count are not loaded (a uniform branch), those past the
    // sequence's count are discarded below
    if (4 * k4 < p.nsplit_ml) {
      const float4 m4 = *reinterpret_cast<const float4 *>(p.ws_m + mbase + 4 * k4);
      const float4 l4 = *reinterpret_cast<const float4 *>(p.ws_l + mbase + 4 * k4);
      mv[4 * k4] = m4.x, mv[4 * k4 + 1] = m4.y, mv[4 * k4 + 2] = m4.z, mv[4 * k4 + 3] = m4.w;
      lv[4 * k4] = l4.x, lv[4 * k4 + 1] = l4.y, lv[4 * k4 + 2] = l4.z, lv[4 * k4 + 3] = l4.w;
    }
  }
#pragma unroll
  for (int k = 0; k < kEager; ++k) {
    if (k < p.nsplit)
      ov[k] = *reinterpret_cast<const float4 *>(p.ws_o + (obase + static_cast<size_t>(k) * p.rows) * DH + c0);
  }
  // keep every load above ahead of the first use of its result (one round trip)
  __builtin_amdgcn_sched_barrier(0);
  bool bad;
  const int S = clamp_prefix(s_raw, p.max_pages, &bad);
  const int npages = (S + kPage - 1) / kPage;
  const int ns = splits_of(npages, p.pages_per_split);
  // a single split was written by the attention kernel. The merge below runs
  // regardless and only the stores are skipped, so that the partials' loads
  // are not deferred behind the prefix length.
  const bool write = live && !(ns == 1 && skip_single);

  float mx = -__builtin_huge_valf();
#pragma unroll
  for (int k = 0; k < kEager; ++k) mx = k < ns ? fmaxf(mx, mv[k]) : mx;
  float den = 0.f, n0 = 0.f, n1 = 0.f, n2 = 0.f, n3 = 0.f;
#pragma unroll
  for (int k = 0; k < kEager; ++k) {
    if (k < ns) {
      const float sc = exp2f(mv[k] - mx);
      den += sc * lv[k];
      n0 += sc * ov[k].x;
      n1 += sc * ov[k].y;
      n2 += sc * ov[k].z;
      n3 += sc * ov[k].w;
    }
  }
  // splits beyond the first 16, merged in the same online form
  for (int s0 = kEager; s0 < ns && live; ++s0) {
    const float m = p.ws_m[mbase + s0], l = p.ws_l[mbase + s0];
    const float4 o = *reinterpret_cast<const float4 *>(p.ws_o + (obase + static_cast<size_t>(s0) * p.rows) * DH + c);
    const float nm = fmaxf(mx, m);
    const float a = exp2f(mx - nm), sc = exp2f(m - nm);
    den = den * a + sc * l;
    n0 = n0 * a + sc * o.x;
    n1 = n1 * a + sc * o.y;
    n2 = n2 * a + sc * o.z;
    n3 = n3 * a + sc * o.w;
    mx = nm;
  }
  if (!write) return;
  const int i = row / p.group, g = row % p.group;
  const int h = kvh * p.group + g;
  T *out = static_cast<T *>(p.out) + ((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH + c;
  const float inv = 1.f / den;
  out[0] = from_f32<T>(n0 * inv);
  out[1] = from_f32<T>(n1 * inv);
  out[2] = from_f32<T>(n2 * inv);
  out[3] = from_f32<T>(n3 * inv);
  if (p.lse && c == 0)
    p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] = (mx + log2f(den)) * 0.69314718055994530942f;
}

// The same merge over the piece records of the matrix-core kernel (one per
// (sequence, KV head, split), piece_record_bytes each): a row's per-split
// {m, l, q} arrive as one 16-byte vector and its outputs as fp16 values
// scaled by q; the records of the first 24 splits are loaded together with
// the prefix length.
template <int DH>
__global__ __launch_bounds__(64) void attn_combine_records_kernel(AttnParams p, int skip_single) {
  const int unit = blockIdx.x;  // b * hkv + kvh
  const int b = unit / p.hkv;
  const int kvh = unit % p.hkv;
  const int row = blockIdx.y * kRowsPerBlock + threadIdx.x / 8;
  const int c = blockIdx.z * kColsPerBlock + 4 * (threadIdx.x % 8);
  const bool live = row < p.rows && c < DH;
  const int r0 = live ? row : 0, c0 = live ? c : 0;
  const size_t stride = static_cast<size_t>(p.piece_stride);
  const uint8_t *rec0 = reinterpret_cast<const uint8_t *>(p.ws_o) +
                        static_cast<size_t>(unit) * p.nsplit * stride;
  const uint8_t *orow = rec0 + (r0 * DH + c0) * 2;
  const uint8_t *mrow = rec0 + static_cast<size_t>(p.rows) * DH * 2 + r0 * 16;

  const int s_raw = p.prefix_len[b];
  f32x4 meta[kEager];
  h16x4 ov[kEager];
#pragma unroll
  for (int k = 0; k < kEager; ++k) {
    if (k < p.nsplit) {  // split slots of the plan (uniform); past the sequence's count: unused
      meta[k] = *reinterpret_cast<const f32x4 *>(mrow + k * stride);
      ov[k] = *reinterpret_cast<const h16x4 *>(orow + k * stride);
    }
  }
  // keep every load above ahead of the first use of its result (one round trip)
  __builtin_amdgcn_sched_barrier(0);
  bool bad;
  const int S = clamp_prefix(s_raw, p.max_pages, &bad);
  const int npages = (S + kPage - 1) / kPage;
  const int ns = splits_of(npages, p.pages_per_split);
  const bool write = live && !(ns == 1 && skip_single);

  // split k: maximum meta[0], sum meta[1], unnormalised output = stored * meta[2]
  float mx = -__builtin_huge_valf();
#pragma unroll
  for (int k = 0; k < kEager; ++k) mx = k < ns ? fmaxf(mx, meta[k][0]) : mx;
  float den = 0.f, n0 = 0.f, n1 = 0.f, n2 = 0.f, n3 = 0.f;
#pragma unroll
  for (int k = 0; k < kEager; ++k) {
    if (k < ns) {
      const float sc = exp2f(meta[k][0] - mx);
      const float wgt = sc * meta[k][2];
      den += sc * meta[k][1];
      n0 += wgt * static_cast<float>(ov[k][0]);
      n1 += wgt * static_cast<float>(ov[k][1]);
      n2 += wgt * static_cast<float>(ov[k][2]);
      n3 += wgt * static_cast<float>(ov[k][3]);
    }
  }
  // splits beyond the first 24, merged in the same online form
  for (int k = kEager; k < ns && live; ++k) {
    const f32x4 mk = *reinterpret_cast<const f32x4 *>(mrow + k * stride);
    const h16x4 o = *reinterpret_cast<const h16x4 *>(orow + k * stride);
    const float nm = fmaxf(mx, mk[0]);
    const float a = exp2f(mx - nm), sc = exp2f(mk[0] - nm);
    const float wgt = sc * mk[2];
    den = den * a + sc * mk[1];
    n0 = n0 * a + wgt * static_cast<float>(o[0]);
    n1 = n1 * a + wgt * static_cast<float>(o[1]);
    n2 = n2 * a + wgt * static_cast<float>(o[2]);
    n3 = n3 * a + wgt * static_cast<float>(o[3]);
    mx = nm;
  }
  if (!write) return;
  const int i = row / p.group, g = row % p.group;
  const int h = kvh * p.group + g;
  bf16_t *out = static_cast<bf16_t *>(p.out) + ((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH + c;
  const float inv = 1.f / den;
  out[0] = f32_to_bf16(n0 * inv);
  out[1] = f32_to_bf16(n1 * inv);
  out[2] = f32_to_bf16(n2 * inv);
  out[3] = f32_to_bf16(n3 * inv);
  if (p.lse && c == 0)
    p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] = (mx + log2f(den)) * 0.69314718055994530942f;
}

template <typename T, int DH>
hipError_t launch_typed(const AttnParams &p, int skip_single, hipStream_t s) {
  dim3 grid(p.batch * p.hkv, (p.rows + kRowsPerBlock - 1) / kRowsPerBlock,
            (DH + kColsPerBlock - 1) / kColsPerBlock);
  return launch_kernel(attn_combine_kernel<T, DH>, grid, dim3(64), s, p, skip_single);
}

template <int DH>
hipError_t launch_records(const AttnParams &p, int skip_single, hipStream_t s) {
  dim3 grid(p.batch * p.hkv, (p.rows + kRowsPerBlock - 1) / kRowsPerBlock,
            (DH + kColsPerBlock - 1) / kColsPerBlock);
  return launch_kernel(attn_combine_records_kernel<DH>, grid, dim3(64), s, p, skip_single);
}

}  // namespace

hipError_t launch_attn_combine_records(const AttnParams &p, int dh, int skip_single,
                                       hipStream_t s) {
  if (dh == 64) return launch_records<64>(p, skip_single, s);
  if (dh == 96) return launch_records<96>(p, skip_single, s);
  return launch_records<128>(p, skip_single, s);
}

hipError_t launch_attn_combine(const AttnParams &p, int dtype, int dh, int skip_single,
                               hipStream_t s) {
  if (dtype == DAS_F32) {
    if (dh == 64) return launch_typed<float, 64>(p, skip_single, s);
    if (dh == 96) return launch_typed<float, 96>(p, skip_single, s);
    return launch_typed<float, 128>(p, skip_single, s);
  }
  if (dh == 64) return launch_typed<bf16_t, 64>(p, skip_single, s);
  if (dh == 96) return launch_typed<bf16_t, 96>(p, skip_single, s);
  return launch_typed<bf16_t, 128>(p, skip_single, s);
}

}  // namespace das
