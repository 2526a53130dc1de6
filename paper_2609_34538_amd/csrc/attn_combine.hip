// Merge of the per-split partial results into the attention output.
//
// Each split s of a (sequence, KV head) left, per query row, an unnormalised
// output O_s, its running maximum m_s (base-2 logit units) and its running
// sum l_s. With M = max_s m_s the joint softmax of Eq. (2) over all splits is
//   O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s,
// and the natural-log normaliser is (M + log2 sum_s 2^(m_s - M) l_s) * ln 2.
// Split 0 always holds the block's diagonal, so M is finite.

#include "das_internal.h"

namespace das {
namespace {

constexpr int kRowsPerBlock = 8;

// One workgroup per (sequence, KV head, group of 8 rows). Each thread owns
// (row, column) outputs and issues the loads of every split's (m, l, O)
// together, so the merge costs one memory round trip.
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p, int skip_single) {
  const int unit = blockIdx.x;  // b * hkv + kvh
  const int b = unit / p.hkv;
  const int kvh = unit % p.hkv;
  bool bad;
  const int S = clamp_prefix(p.prefix_len[b], p.max_pages, &bad);
  const int npages = (S + kPage - 1) / kPage;
  int ns = (npages + p.pages_per_split - 1) / p.pages_per_split;
  if (ns < 1) ns = 1;
  if (ns == 1 && skip_single) return;  // the attention kernel wrote it
  const size_t base_row = (static_cast<size_t>(unit) * p.nsplit) * p.rows;
  T *out = static_cast<T *>(p.out);
  const int row0 = blockIdx.y * kRowsPerBlock;
  const int nrows = min(kRowsPerBlock, p.rows - row0);

  for (int e = threadIdx.x; e < nrows * DH; e += blockDim.x) {
    const int row = row0 + e / DH, c = e % DH;
    float mx = -__builtin_huge_valf(), num = 0.f, den = 0.f;
    constexpr int CH = 8;
    for (int s0 = 0; s0 < ns; s0 += CH) {
      float mv[CH], lv[CH], ov[CH];
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const int s = s0 + k;
        const size_t r = base_row + static_cast<size_t>(s < ns ? s : 0) * p.rows + row;
        mv[k] = s < ns ? p.ws_m[r] : -__builtin_huge_valf();
        lv[k] = p.ws_l[r];
        ov[k] = p.ws_o[r * DH + c];
      }
      float cm = mx;
#pragma unroll
      for (int k = 0; k < CH; ++k) cm = fmaxf(cm, mv[k]);
      const float rescale = exp2f(mx - cm);  // 0 on the first chunk (mx = -inf)
      num *= rescale;
      den *= rescale;
#pragma unroll
      for (int k = 0; k < CH; ++k) {
        const float sc = exp2f(mv[k] - cm);
        num += sc * ov[k];
        den += sc * lv[k];
      }
      mx = cm;
    }
    const int i = row / p.group, g = row % p.group;
    const int h = kvh * p.group + g;
    out[((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH + c] = from_f32<T>(num / den);
    if (p.lse && c == 0)
      p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] = (mx + log2f(den)) * 0.69314718055994530942f;
  }
}

template <typename T, int DH>
hipError_t launch_typed(const AttnParams &p, int skip_single, hipStream_t s) {
  dim3 grid(p.batch * p.hkv, (p.rows + kRowsPerBlock - 1) / kRowsPerBlock);
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), grid, dim3(256), 0, s, p, skip_single);
  return hipGetLastError();
}

}  // namespace

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
