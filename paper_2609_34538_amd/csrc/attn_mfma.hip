// Matrix-core (MFMA) policy-attention kernel for bf16 caches (Eq. (2)-(3)).
//
// Persistent one-wave workers. The work of a call is cut into chunks =
// (sequence, KV head, row tile of 16 * NQ query rows, prefix split of up to
// pages_per_split pages); split 0 of every (sequence, head, row tile) also
// carries the draft block. Chunks are enumerated with every full split first
// and the shorter last splits after them, and worker r takes chunks r, r + W,
// r + 2W, ... (W = number of workers, a multiple of 8): every worker gets
// about the same number of full chunks. Workgroups are dealt to the 8 XCDs
// round-robin, so chunk c runs on XCD c mod 8 and even a call with fewer
// chunks than workers spreads over every XCD. Inside each run of 8 splits
// the row tiles of one split are numbered 8 apart, which puts them on one
// XCD, where they share its L2.
//
// Each worker streams the 32-token tiles of its chunks (two per prefix page,
// then the draft block's), one chunk after the other, through a private
// ring of NB LDS slots filled by the direct-to-LDS loads of gfx950
// (global_load_lds_dwordx4), up to NB tiles ahead of the tile being computed
// and across chunk boundaries; a chunk's Q fragments go into one of two LDS
// buffers the same way when the stream enters the chunk. The worker waits on
// its own vector-memory counter for the data it reads. Load addresses are a
// uniform base (page, fragment) plus one per-lane offset, so issuing a tile
// costs no per-lane address arithmetic. Chunk descriptors and page ids are
// decoded a batch of chunks at a time into registers.
//
// Both products run on v_mfma_f32_16x16x32_bf16 with the key/value tile as
// the A operand, so softmax probabilities never leave registers:
//   S^T (tokens x rows) = K_tile (tokens x dh) . Q^T (dh x rows)
//   O^T (dh x rows)    += V^T_tile (dh x tokens) . P^T (tokens x rows)
// MFMA 16x16x32 bf16 lane layout (lane l, n = l % 16, g = l / 16):
//   A[m][k]: lane holds m = n, k = 8g..8g+7   B[k][n]: k = 8g..8g+7, n
//   C[m][n]: lane holds m = 4g..4g+3, n
// The 16 token slots of each S^T tile are a permutation of the tile's tokens
// chosen so that the C fragments of the tile's two S^T halves hold, per lane,
// the 8 consecutive tokens 8g .. 8g + 7; those are exactly the k slots of the
// P^T fragment of the P.V product, and the matching V^T fragment is one
// contiguous 16-byte load from the token-grouped value page ([8][dh][8]);
// a 32-token tile of that page is one contiguous block. The draft block's
// values are token-major; their V^T fragments are gathered from LDS.
//
// A chunk ends by writing its (m, l, O) partial to the workspace for the
// combine kernel, or, when its sequence has a single split, the normalised
// output. Query rows of a row tile: row = i * G + g (block position i,
// head kvh * G + g). Logits are scaled into base-2 units after the product.

#include <atomic>

#include "das_internal.h"

namespace das {
namespace {

constexpr int kMaxDevices = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kFragBytes = 64 * 16;  // one 16-byte fragment per lane
constexpr int kBatch = 8;            // chunks decoded at a time (8 fields each)
constexpr int kMaxSeqBlocks = 64;    // sequences are scanned 64 at a time

// 16 bytes per lane, global -> LDS at lds + 16 * lane (lds wave-uniform).
__device__ __forceinline__ void dma16(const void *src, uint8_t *lds) {
  __builtin_amdgcn_global_load_lds((__attribute__((address_space(1))) void *)(src),
                                   (__attribute__((address_space(3))) void *)(lds), 16, 0, 0);
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

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

template <int DH, int NQ, int NB_>
struct Geo {
  static constexpr int KS = DH / 32;       // k steps of Q K^T
  static constexpr int DT = DH / 16;       // head-dim tiles of P V
  static constexpr int NF = 2 * KS + DT;   // fragments (loads) per 32-token tile
  static constexpr int SLOT = NF * kFragBytes;
  static constexpr int NB = NB_;           // ring depth
  static constexpr int QF = NQ * KS;       // Q fragments of a row tile
  static constexpr int LDS = NB * SLOT + 2 * QF * kFragBytes + kBatch * 64 * 4 +
                             2 * kMaxSeqBlocks * 4;
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
template <int DH, int NQ, typename Hook>
__device__ __forceinline__ void compute_tile(State<DH, NQ> &st, const u32x4 (&kf)[2][DH / 32],
                                             const u32x4 (&vf)[DH / 16],
                                             const u32x4 (&qf)[NQ][DH / 32],
                                             const int (&cap)[NQ], int limit, bool full,
                                             float scale, int lg, Hook &&hook) {
  u16x8 pf[NQ];
  float alpha[NQ];
  bool moved = false;
  f32x4 sacc[NQ][2];
  hook(0);
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      sacc[qt][e] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < DH / 32; ++ks)
        sacc[qt][e] = mfma16x16x32(kf[e][ks], qf[qt][ks], sacc[qt][e]);
    }
  }
  hook(1);
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    float x[2][4];
    float mx = kNegInf;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int t = 8 * lg + 4 * e + v;
        const bool vis = full || ((t < limit) & (t <= cap[qt]));
        x[e][v] = vis ? sacc[qt][e][v] * scale : kNegInf;
        mx = fmaxf(mx, x[e][v]);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mnew = fmaxf(st.m[qt], mx);
    const float muse = mnew == kNegInf ? 0.f : mnew;
    alpha[qt] = __builtin_amdgcn_exp2f(st.m[qt] - muse);
    moved |= alpha[qt] != 1.f;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float pv = __builtin_amdgcn_exp2f(x[e][v] - muse);
        psum += pv;
        pf[qt][4 * e + v] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(pv));
      }
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    st.l[qt] = st.l[qt] * alpha[qt] + psum;
    st.m[qt] = mnew;
  }
  hook(2);
  // rescale the accumulators only when some row's maximum moved
  if (__builtin_amdgcn_ballot_w64(moved) != 0) {
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt)
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) st.o[qt][dt] *= alpha[qt];
  }
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) {
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt)
      st.o[qt][dt] = mfma16x16x32(vf[dt], __builtin_bit_cast(u32x4, pf[qt]), st.o[qt][dt]);
  }
}

// Chunk counts of one block of 64 sequences (lane j holds sequence 64k + j).
struct SeqBlock {
  int k;            // block index held (-1: none)
  int S;            // this lane's clamped prefix length
  int npages;
  int nfull;        // full splits x units
  int npart;        // (1 if the last split is shorter or the prefix is empty) x units
  int inclF, inclP; // inclusive prefix sums over the block's lanes
};

// Fields of a decoded chunk, lane 8j + f of the descriptor register.
enum { F_B = 0, F_KVH, F_RT, F_SPLIT, F_PG0, F_NPG, F_S, F_NSB };

// DIRECT: one workgroup per chunk (grid = every possible chunk, n_workers =
// grid size); the chunk is decoded from the workgroup id, so the prefix
// length, the chunk's page ids and its Q rows are fetched in one round trip.
// Otherwise persistent workers scan the prefix lengths and walk their chunks.
template <int DH, int NQ, int NB, bool DIRECT>
__global__ __launch_bounds__(64) void attn_mfma_kernel(AttnParams p, int n_rt, int n_workers) {
  using G = Geo<DH, NQ, NB>;
  constexpr int KS = G::KS;
  constexpr int DT = G::DT;
  constexpr int NF = G::NF;
  constexpr int ROWS = 16 * NQ;
  __shared__ __attribute__((aligned(16))) uint8_t ring[NB * G::SLOT];
  __shared__ __attribute__((aligned(16))) uint8_t qbuf[2][G::QF * kFragBytes];
  __shared__ int pid[kBatch][64];      // page ids of each decoded chunk
  __shared__ int blkF[kMaxSeqBlocks];  // full-split chunks of each sequence block
  __shared__ int blkP[kMaxSeqBlocks];  // last-split chunks of each sequence block

  const int lane = threadIdx.x;
  const int ln = lane & 15;
  const int lg = lane >> 4;
  const int rank = blockIdx.x;  // runs on XCD rank mod 8
  const int pps = p.pages_per_split;
  const int units = p.hkv * n_rt;  // chunks per split of one sequence
  const int nblocks = (p.batch + 63) >> 6;
  const int nblk = (p.w + 31) >> 5;  // draft-block tiles of a split-0 chunk

  SeqBlock sb;
  sb.k = -1;
  auto load_block = [&](int k) {
    const int b = 64 * k + lane;
    const bool live = b < p.batch;
    const int s_raw = live ? p.prefix_len[b] : 0;
    bool bad;
    const int S = clamp_prefix(s_raw, p.max_pages, &bad);
    if (bad && live && rank == 0) report_error(p.dev_error, DAS_DEVERR_PREFIX);
    sb.k = k;
    sb.S = S;
    sb.npages = (S + kPage - 1) / kPage;
    sb.nfull = live ? (sb.npages / pps) * units : 0;
    sb.npart = live ? ((sb.npages % pps) != 0 || sb.npages == 0 ? units : 0) : 0;
    int f = sb.nfull, q = sb.npart;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int fu = __shfl_up(f, o, 64), qu = __shfl_up(q, o, 64);
      if (lane >= o) {
        f += fu;
        q += qu;
      }
    }
    sb.inclF = f;
    sb.inclP = q;
  };

  int totF = 0, totP = 0;
  int my_chunks = 1;
  if constexpr (!DIRECT) {
  for (int k = 0; k < nblocks; ++k) {
    load_block(k);
    const int bf = __shfl(sb.inclF, 63, 64), bp = __shfl(sb.inclP, 63, 64);
    if (lane == 0) {
      blkF[k] = bf;
      blkP[k] = bp;
    }
    totF += bf;
    totP += bp;
  }
  const int total = totF + totP;
  my_chunks = rank < total ? (total - rank + n_workers - 1) / n_workers : 0;
  if (my_chunks == 0) return;
  }

  // Batch of decoded chunks: descv lane 8j + f = field f of chunk j, and
  // pid[j][i] = page id of the chunk's i-th page. The descriptors are
  // computed first and the page-table loads of the whole batch issued after
  // them, so the batch costs one memory round trip.
  int descv = 0;
  auto field = [&](int j, int f) { return __builtin_amdgcn_readlane(descv, 8 * j + f); };
  auto decode_batch = [&](int first, int count) {
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (j >= count) continue;
      const int c = rank + (first + j) * n_workers;
      const bool phase2 = c >= totF;
      int rem = phase2 ? c - totF : c;
      // chunk number -> (split group, row tile): in each complete run of 8
      // groups of n_rt row tiles, row tile rt of group 8k + x is number
      // 8 n_rt k + 8 rt + x
      {
        const int span = 8 * n_rt;
        const int runs = ((phase2 ? totP : totF) / n_rt) >> 3;
        if (rem < runs * span) {
          const int k = rem / span, x = rem % span;
          rem = (8 * k + (x & 7)) * n_rt + (x >> 3);
        }
      }
      int k = 0;
      while (k < nblocks - 1) {
        const int n = phase2 ? blkP[k] : blkF[k];
        if (rem < n) break;
        rem -= n;
        ++k;
      }
      if (sb.k != k) load_block(k);
      const int incl = phase2 ? sb.inclP : sb.inclF;
      const int own = phase2 ? sb.npart : sb.nfull;
      const unsigned long long m = __ballot(incl > rem);
      const int lb = __builtin_ctzll(m);
      const int local = rem - (__shfl(incl, lb, 64) - __shfl(own, lb, 64));
      const int b = 64 * k + lb;
      const int S = __shfl(sb.S, lb, 64);
      const int npages = __shfl(sb.npages, lb, 64);
      const int full = npages / pps;
      const int split = phase2 ? full : local / units;
      const int u = local % units;
      const int pg0 = split * pps;
      const int npg = max(0, min(pps, npages - pg0));
      const int nsb = max(1, (npages + pps - 1) / pps);
      const int d = lane - 8 * j;
      descv = d == F_B ? b : descv;
      descv = d == F_KVH ? u / n_rt : descv;
      descv = d == F_RT ? u % n_rt : descv;
      descv = d == F_SPLIT ? split : descv;
      descv = d == F_PG0 ? pg0 : descv;
      descv = d == F_NPG ? npg : descv;
      descv = d == F_S ? S : descv;
      descv = d == F_NSB ? nsb : descv;
    }
    int pages[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      pages[j] = 0;
      const int b = uni(field(j, F_B)), pg0 = uni(field(j, F_PG0));
      const int npg = j < count ? uni(field(j, F_NPG)) : 0;
      if (lane < npg) pages[j] = p.block_table[static_cast<size_t>(b) * p.max_pages + pg0 + lane];
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) pid[j][lane] = pages[j];
  };
  auto pages_of = [&](int j) { return pid[j][lane]; };

  const char *kl = static_cast<const char *>(p.k_layer);
  const char *vl = static_cast<const char *>(p.v_layer);
  const size_t head_bytes = static_cast<size_t>(p.num_pages) * kPage * DH * 2;
  const size_t tok_bytes = static_cast<size_t>(p.hkv) * DH * 2;  // block row stride
  // per-lane byte offsets of the fragments inside a page: key token slot
  // 8(n/4) + n%4 (plus a uniform part), column 8g; value token group g of
  // the tile, head dim n
  const uint32_t lane_k = ((8 * (ln >> 2) + (ln & 3)) * DH + 8 * lg) * 2;
  const uint32_t lane_v = (lg * DH + ln) * 16;

  // Issue cursor: batch chunk ij, next tile it of its ntile (= 2 npg page
  // tiles, then nblk block tiles on split 0); n_issued tiles so far. Compute
  // cursor: chunk cj, n_done tiles consumed. Q of batch chunk j sits in
  // qbuf[j & 1].
  int batch_base = 0, batch_len = 0;
  int ij = -1, it = 0, i_ntile = 0, i_npg2 = 0, i_kvh = 0, i_b = 0;
  int i_pages = 0;
  int n_issued = 0;
  int cj = 0, n_done = 0;
  int q_tiles0 = 0, q_tiles1 = 0;  // n_issued when each Q buffer was loaded

  auto issue_q = [&](int j, int b, int kvh, int rt) {
    uint8_t *qb = qbuf[j & 1];
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      // rows past the last are clamped; their outputs are never written
      const int row = min(rt * ROWS + qt * 16 + ln, p.rows - 1);
      const int i = row / p.group, g = row % p.group;
      const bf16_t *qrow = static_cast<const bf16_t *>(p.q) +
                           ((static_cast<size_t>(b) * p.w + i) * p.hq + kvh * p.group + g) * DH;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) dma16(qrow + 32 * ks + 8 * lg, qb + (qt * KS + ks) * kFragBytes);
    }
    if (j & 1) q_tiles1 = n_issued;
    else q_tiles0 = n_issued;
  };

  // Put one more tile in the ring if there is room, entering the next chunk
  // when the current one is exhausted (at most one chunk ahead of the compute
  // cursor, so both Q buffers stay valid).
  auto try_issue = [&]() {
    while (true) {
      if (ij >= 0 && it < i_ntile) {
        if (n_issued - n_done >= NB) return;
        uint8_t *slot = ring + (n_issued % NB) * G::SLOT;
        if (it < i_npg2) {
          const int page = __builtin_amdgcn_readlane(i_pages, it >> 1);
          const bool ok = page >= 0 && page < p.num_pages;
          if (!ok) report_error(p.dev_error, DAS_DEVERR_PAGE);
          const size_t off = i_kvh * head_bytes + static_cast<size_t>(ok ? page : 0) * kPage * DH * 2;
          const int u = it & 1;
          const char *kb = kl + off + (32 * u) * DH * 2;
          const char *vb = vl + off + 64 * DH * u;  // token groups 4u .. 4u + 3
#pragma unroll
          for (int e = 0; e < 2; ++e)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              dma16(kb + (4 * e * DH + 32 * ks) * 2 + lane_k, slot + (e * KS + ks) * kFragBytes);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            dma16(vb + 256 * dt + lane_v, slot + (2 * KS + dt) * kFragBytes);
        } else {
          // draft block tile u: key fragments by token slot, value rows raw
          const int u = it - i_npg2;
          const char *kb = static_cast<const char *>(p.kb) +
                           (static_cast<size_t>(i_b) * p.w * p.hkv + i_kvh) * DH * 2;
          const char *vb = static_cast<const char *>(p.vb) +
                           (static_cast<size_t>(i_b) * p.w * p.hkv + i_kvh) * DH * 2;
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const int tok = min(32 * u + 8 * (ln >> 2) + 4 * e + (ln & 3), p.w - 1);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              dma16(kb + tok * tok_bytes + (32 * ks + 8 * lg) * 2, slot + (e * KS + ks) * kFragBytes);
          }
#pragma unroll
          for (int f = 0; f < DT; ++f) {
            const int o = f * kFragBytes + 16 * lane;  // byte in the [32][DH] half
            const int tok = min(32 * u + o / (2 * DH), p.w - 1);
            dma16(vb + tok * tok_bytes + o % (2 * DH), slot + (2 * KS + f) * kFragBytes);
          }
        }
        ++n_issued;
        ++it;
        return;
      }
      const int nj = ij + 1;
      if (nj >= batch_len || nj > cj + 1) return;
      ij = nj;
      it = 0;
      i_b = uni(field(nj, F_B));
      i_kvh = uni(field(nj, F_KVH));
      i_npg2 = 2 * uni(field(nj, F_NPG));
      i_ntile = i_npg2 + (uni(field(nj, F_SPLIT)) == 0 ? nblk : 0);
      i_pages = pages_of(nj);
      issue_q(nj, i_b, i_kvh, uni(field(nj, F_RT)));
    }
  };

  // The same issue split in three parts (key fragments of each S^T half,
  // then the values) so the loads of the next tile can be spread over the
  // computation of the current one.
  bool s_have = false;
  bool s_blk = false;
  const char *s_kb = nullptr, *s_vb = nullptr;
  uint8_t *s_slot = nullptr;
  int s_u = 0;
  auto stage_begin = [&]() {
    s_have = false;
    while (true) {
      if (ij >= 0 && it < i_ntile) {
        if (n_issued - n_done >= NB) return;
        s_have = true;
        s_slot = ring + (n_issued % NB) * G::SLOT;
        s_blk = it >= i_npg2;
        if (!s_blk) {
          const int page = __builtin_amdgcn_readlane(i_pages, it >> 1);
          const bool ok = page >= 0 && page < p.num_pages;
          if (!ok) report_error(p.dev_error, DAS_DEVERR_PAGE);
          const size_t off = i_kvh * head_bytes + static_cast<size_t>(ok ? page : 0) * kPage * DH * 2;
          s_u = it & 1;
          s_kb = kl + off + (32 * s_u) * DH * 2;
          s_vb = vl + off + 64 * DH * s_u;
        } else {
          s_u = it - i_npg2;
          s_kb = static_cast<const char *>(p.kb) + (static_cast<size_t>(i_b) * p.w * p.hkv + i_kvh) * DH * 2;
          s_vb = static_cast<const char *>(p.vb) + (static_cast<size_t>(i_b) * p.w * p.hkv + i_kvh) * DH * 2;
        }
        return;
      }
      const int nj = ij + 1;
      if (nj >= batch_len || nj > cj + 1) return;
      ij = nj;
      it = 0;
      i_b = uni(field(nj, F_B));
      i_kvh = uni(field(nj, F_KVH));
      i_npg2 = 2 * uni(field(nj, F_NPG));
      i_ntile = i_npg2 + (uni(field(nj, F_SPLIT)) == 0 ? nblk : 0);
      i_pages = pages_of(nj);
      issue_q(nj, i_b, i_kvh, uni(field(nj, F_RT)));
    }
  };
  auto stage_part = [&](int part) {
    if (!s_have) return;
    if (part < 2) {
      const int e = part;
      if (!s_blk) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          dma16(s_kb + (4 * e * DH + 32 * ks) * 2 + lane_k, s_slot + (e * KS + ks) * kFragBytes);
      } else {
        const int tok = min(32 * s_u + 8 * (ln >> 2) + 4 * e + (ln & 3), p.w - 1);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          dma16(s_kb + tok * tok_bytes + (32 * ks + 8 * lg) * 2, s_slot + (e * KS + ks) * kFragBytes);
      }
    } else {
      if (!s_blk) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          dma16(s_vb + 256 * dt + lane_v, s_slot + (2 * KS + dt) * kFragBytes);
      } else {
#pragma unroll
        for (int f = 0; f < DT; ++f) {
          const int o = f * kFragBytes + 16 * lane;  // byte in the [32][DH] half
          const int tok = min(32 * s_u + o / (2 * DH), p.w - 1);
          dma16(s_vb + tok * tok_bytes + o % (2 * DH), s_slot + (2 * KS + f) * kFragBytes);
        }
      }
      ++n_issued;
      ++it;
      s_have = false;
    }
  };

  auto start_batch = [&]() {
    batch_len = min(kBatch, my_chunks - batch_base);
    decode_batch(batch_base, batch_len);
    ij = -1;
    it = 0;
    cj = 0;
    for (int k = 0; k < NB; ++k) try_issue();
  };

  if constexpr (DIRECT) {
    // chunk number -> (split group, row tile) as in the persistent order;
    // group = (b * nsplit + split) * hkv + kvh
    int grp, rt;
    {
      const int c = blockIdx.x, span = 8 * n_rt, runs = (n_workers / n_rt) >> 3;
      if (c < runs * span) {
        grp = 8 * (c / span) + (c % span & 7);
        rt = (c % span) >> 3;
      } else {
        grp = c / n_rt;
        rt = c % n_rt;
      }
    }
    const int kvh = grp % p.hkv;
    const int split = (grp / p.hkv) % p.nsplit;
    const int b = grp / p.hkv / p.nsplit;
    const int pg0 = split * pps;
    // one round trip: prefix length, this split's page ids, Q rows
    const int s_raw = p.prefix_len[b];
    int page = 0;
    if (lane < pps && pg0 + lane < p.max_pages)
      page = p.block_table[static_cast<size_t>(b) * p.max_pages + pg0 + lane];
    issue_q(0, b, kvh, rt);
    bool bad;
    const int S = clamp_prefix(s_raw, p.max_pages, &bad);
    if (bad && split == 0 && kvh == 0 && rt == 0 && lane == 0)
      report_error(p.dev_error, DAS_DEVERR_PREFIX);
    const int npages = (S + kPage - 1) / kPage;
    const int nsb = max(1, (npages + pps - 1) / pps);
    if (split >= nsb) {
      wait_vmcnt<0>();  // the Q rows land in LDS before the workgroup ends
      return;
    }
    const int npg = max(0, min(pps, npages - pg0));
    descv = lane == F_B ? b : descv;
    descv = lane == F_KVH ? kvh : descv;
    descv = lane == F_RT ? rt : descv;
    descv = lane == F_SPLIT ? split : descv;
    descv = lane == F_PG0 ? pg0 : descv;
    descv = lane == F_NPG ? npg : descv;
    descv = lane == F_S ? S : descv;
    descv = lane == F_NSB ? nsb : descv;
    pid[0][lane] = page;
    batch_len = 1;
    ij = 0;
    it = 0;
    cj = 0;
    i_b = b;
    i_kvh = kvh;
    i_npg2 = 2 * npg;
    i_ntile = i_npg2 + (split == 0 ? nblk : 0);
    i_pages = page;
    for (int k = 0; k < NB; ++k) try_issue();
  } else {
    start_batch();
  }
  while (true) {
    if (cj >= batch_len) {
      batch_base += batch_len;
      if (batch_base >= my_chunks) break;
      wait_vmcnt<0>();  // ring and Q buffers idle before the next batch
      start_batch();
      continue;
    }
    while (ij < cj) try_issue();  // enter this chunk (loads its Q)
    const int b = uni(field(cj, F_B)), kvh = uni(field(cj, F_KVH)), rt = uni(field(cj, F_RT));
    const int split = uni(field(cj, F_SPLIT)), pg0 = uni(field(cj, F_PG0));
    const int npg = uni(field(cj, F_NPG)), S = uni(field(cj, F_S)), nsb = uni(field(cj, F_NSB));
    const int c_pages = pages_of(cj);
    const int ntile = 2 * npg + (split == 0 ? nblk : 0);
    wait_tiles<NF>(n_issued - ((cj & 1) ? q_tiles1 : q_tiles0));
    u32x4 qf[NQ][KS];
    int cap_blk[NQ];
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      cap_blk[qt] = (rt * ROWS + qt * 16 + ln) / p.group;  // block position i of the row
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[qt][ks] = *reinterpret_cast<const u32x4 *>(qbuf[cj & 1] + (qt * KS + ks) * kFragBytes + 16 * lane);
    }
    State<DH, NQ> st;
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      st.m[qt] = kNegInf;
      st.l[qt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) st.o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    for (int t = 0; t < ntile; ++t) {
      wait_tiles<NF>(n_issued - n_done - 1);
      const uint8_t *slot = ring + (n_done % NB) * G::SLOT;
      ++n_done;
      u32x4 kf[2][KS], vf[DT];
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          kf[e][ks] = *reinterpret_cast<const u32x4 *>(slot + (e * KS + ks) * kFragBytes + 16 * lane);
      int cap[NQ];
      int limit;
      bool full;
      if (t < 2 * npg) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          vf[dt] = *reinterpret_cast<const u32x4 *>(slot + (2 * KS + dt) * kFragBytes + 16 * lane);
        const int page = __builtin_amdgcn_readlane(c_pages, t >> 1);
        const bool ok = page >= 0 && page < p.num_pages;
        limit = ok ? min(32, S - (pg0 + (t >> 1)) * kPage - 32 * (t & 1)) : 0;
        full = limit >= 32;
#pragma unroll
        for (int qt = 0; qt < NQ; ++qt) cap[qt] = 0x7fffffff;
      } else {
        // block values are token-major [32][DH] in the slot: gather V^T
        const int u = t - 2 * npg;
        const uint16_t *raw = reinterpret_cast<const uint16_t *>(slot + 2 * KS * kFragBytes);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          u16x8 v8;
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) v8[jj] = raw[(8 * lg + jj) * DH + 16 * dt + ln];
          vf[dt] = __builtin_bit_cast(u32x4, v8);
        }
        limit = p.w - 32 * u;
        full = false;
#pragma unroll
        for (int qt = 0; qt < NQ; ++qt) cap[qt] = cap_blk[qt] - 32 * u;
      }
      // the slot's fragments are in registers before it is refilled
      __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)
      stage_begin();
      compute_tile<DH, NQ>(st, kf, vf, qf, cap, limit, full, p.scale_log2, lg,
                           [&](int k) { stage_part(k); });
    }
    ++cj;
    for (int k = 0; k < NB; ++k) try_issue();  // keep the stream going into the next chunk

    // Chunk result. Lane holds head dims 16dt + 4g .. +3 of row n of tile qt.
    const size_t prow0 = ((static_cast<size_t>(b) * p.hkv + kvh) * p.nsplit + split) * p.rows;
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      const int row = rt * ROWS + qt * 16 + ln;
      if (row >= p.rows) continue;
      if (nsb == 1) {
        const float inv = 1.f / st.l[qt];
        const int i = row / p.group, h = kvh * p.group + row % p.group;
        bf16_t *orow = static_cast<bf16_t *>(p.out) +
                       ((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const f32x4 o = st.o[qt][dt];
          u32x2 packed;
          packed[0] = static_cast<uint32_t>(f32_to_bf16(o[0] * inv)) |
                      (static_cast<uint32_t>(f32_to_bf16(o[1] * inv)) << 16);
          packed[1] = static_cast<uint32_t>(f32_to_bf16(o[2] * inv)) |
                      (static_cast<uint32_t>(f32_to_bf16(o[3] * inv)) << 16);
          *reinterpret_cast<u32x2 *>(orow + 16 * dt + 4 * lg) = packed;
        }
        if (lg == 0 && p.lse)
          p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] =
              (st.m[qt] + log2f(st.l[qt])) * 0.69314718055994530942f;
      } else {
        float *orow = p.ws_o + (prow0 + row) * DH;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) *reinterpret_cast<f32x4 *>(orow + 16 * dt + 4 * lg) = st.o[qt][dt];
        if (lg == 0) {
          p.ws_m[prow0 + row] = st.m[qt] == kNegInf ? 0.f : st.m[qt];
          p.ws_l[prow0 + row] = st.l[qt];
        }
      }
    }
  }
}

// Workers resident per compute unit, from the LDS each one needs.
template <int DH, int NQ, int NB>
constexpr int workers_per_cu() {
  constexpr int n = (160 * 1024) / Geo<DH, NQ, NB>::LDS;
  return n > 8 ? 8 : (n < 1 ? 1 : n);
}

template <int DH, int NQ, int NB>
hipError_t launch_typed(const AttnParams &p, int n_cu, int sched, hipStream_t s) {
  const int n_rt = (p.rows + 16 * NQ - 1) / (16 * NQ);
  const int workers = n_cu * workers_per_cu<DH, NQ, NB>();
  // every possible chunk (the table width bounds the splits of a sequence)
  const long slots = static_cast<long>(p.batch) * p.hkv * p.nsplit * n_rt;
  const bool per_chunk =
      sched == DAS_SCHED_PER_CHUNK || (sched == DAS_SCHED_AUTO && slots <= workers);
  if (per_chunk) {
    hipLaunchKernelGGL((attn_mfma_kernel<DH, NQ, NB, true>), dim3(static_cast<int>(slots)),
                       dim3(64), 0, s, p, n_rt, static_cast<int>(slots));
  } else {
    hipLaunchKernelGGL((attn_mfma_kernel<DH, NQ, NB, false>), dim3(workers), dim3(64), 0, s, p,
                       n_rt, workers);
  }
  return hipGetLastError();
}

template <int DH>
hipError_t launch_dh(const AttnParams &p, int n_cu, int sched, hipStream_t s) {
  if (p.rows <= 16) return launch_typed<DH, 1, 2>(p, n_cu, sched, s);
  return launch_typed<DH, 2, 2>(p, n_cu, sched, s);
}

}  // namespace

// Compute units of each device, queried once (0 = not yet known).
std::atomic<int> g_cu_count[kMaxDevices];

hipError_t launch_attn_mfma(const AttnParams &p, int dh, int sched, hipStream_t s) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return hipErrorInvalidDevice;
  int n_cu = dev < kMaxDevices ? g_cu_count[dev].load(std::memory_order_relaxed) : 0;
  if (n_cu == 0) {
    if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n_cu < 1)
      return hipErrorInvalidDevice;
    n_cu = (n_cu + 7) / 8 * 8;  // the worker ranking assumes a multiple of 8
    if (dev < kMaxDevices) g_cu_count[dev].store(n_cu, std::memory_order_relaxed);
  }
  if (dh == 64) return launch_dh<64>(p, n_cu, sched, s);
  if (dh == 96) return launch_dh<96>(p, n_cu, sched, s);
  return launch_dh<128>(p, n_cu, sched, s);
}

}  // namespace das
