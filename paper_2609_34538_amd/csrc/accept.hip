// Greedy verification of a block (Sec. 3.4): proposals are accepted in order
// while they equal the verifier's predictions; the first mismatch emits the
// prediction in its place and ends the block. The number of retained
// verifier inputs, min(accepted + 1, w), is written where das_kv_append reads
// its commit counts, so the commit follows on the device.
//
// One wave per sequence, lane i holding position i (w <= 64): the accepted
// count is the length of the leading run of matches among the first m
// positions, found with one ballot.

#include "das_internal.h"

namespace das {
namespace {

constexpr int kSeqPerBlock = 4;

__global__ __launch_bounds__(64 * kSeqPerBlock) void greedy_accept_kernel(AcceptParams p) {
  const int lane = threadIdx.x % 64;
  const int b = blockIdx.x * kSeqPerBlock + threadIdx.x / 64;
  if (b >= p.batch) return;  // whole wave
  const int w = p.w;
  int m = w;
  if (p.tested) {
    const int raw = p.tested[b];
    m = min(max(raw, 0), w);
    if (raw != m && lane == 0) report_error(p.dev_error, DAS_DEVERR_TESTED);
  }
  const size_t row = static_cast<size_t>(b) * w;
  int y = 0, yhat = 0;
  if (lane < w) {
    y = p.proposals[row + lane];
    yhat = p.target_pred[row + lane];
  }
  const bool match = lane < m && y == yhat;
  // leading matches: index of the first lane that does not match
  const unsigned long long miss = ~__ballot(match);
  const int a = min(miss ? static_cast<int>(__builtin_ctzll(miss)) : 64, m);
  const int keep = min(a + 1, w);
  if (lane == 0) {
    p.accepted[b] = a;
    p.num_keep[b] = keep;
    if (p.num_emitted) p.num_emitted[b] = keep;
  }
  if (p.emitted && lane < keep) p.emitted[row + lane] = lane < a ? y : yhat;
}

}  // namespace

hipError_t launch_greedy_accept(const AcceptParams &p, hipStream_t s) {
  const int blocks = (p.batch + kSeqPerBlock - 1) / kSeqPerBlock;
  return launch_kernel(greedy_accept_kernel, dim3(blocks), dim3(64 * kSeqPerBlock), s, p);
}

}  // namespace das
