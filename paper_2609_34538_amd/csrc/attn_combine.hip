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

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnParams p) {
  const int unit = blockIdx.x;  // b * hkv + kvh
  const int b = unit / p.hkv;
  const int kvh = unit % p.hkv;
  bool bad;
  const int S = clamp_prefix(p.prefix_len[b], p.max_pages, &bad);
  const int npages = (S + kPage - 1) / kPage;
  int ns = (npages + p.pages_per_split - 1) / p.pages_per_split;
  if (ns < 1) ns = 1;
  const size_t base_row = (static_cast<size_t>(unit) * p.nsplit) * p.rows;
  T *out = static_cast<T *>(p.out);

  for (int row = blockIdx.y; row < p.rows; row += gridDim.y) {
    float mx = -__builtin_huge_valf();
    for (int s = 0; s < ns; ++s) mx = fmaxf(mx, p.ws_m[base_row + static_cast<size_t>(s) * p.rows + row]);
    float den = 0.f;
    for (int s = 0; s < ns; ++s) {
      const size_t r = base_row + static_cast<size_t>(s) * p.rows + row;
      den += exp2f(p.ws_m[r] - mx) * p.ws_l[r];
    }
    const float inv = 1.f / den;
    const int i = row / p.group, g = row % p.group;
    const int h = kvh * p.group + g;
    for (int c = threadIdx.x; c < DH; c += blockDim.x) {
      float num = 0.f;
      for (int s = 0; s < ns; ++s) {
        const size_t r = base_row + static_cast<size_t>(s) * p.rows + row;
        num += exp2f(p.ws_m[r] - mx) * p.ws_o[r * DH + c];
      }
      out[((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH + c] = from_f32<T>(num * inv);
    }
    if (p.lse && threadIdx.x == 0)
      p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] =
          (mx + log2f(den)) * 0.69314718055994530942f;
  }
}

template <typename T, int DH>
hipError_t launch_typed(const AttnParams &p, hipStream_t s) {
  const int rows_per_grid = p.rows < 64 ? p.rows : 64;
  dim3 grid(p.batch * p.hkv, rows_per_grid);
  hipLaunchKernelGGL((attn_combine_kernel<T, DH>), grid, dim3(DH <= 64 ? 64 : 128), 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_combine(const AttnParams &p, int dtype, int dh, hipStream_t s) {
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
