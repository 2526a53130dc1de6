// Matrix-core (MFMA) policy-attention kernel for bf16 caches (Eq. (2)-(3)).
//
// One wave per chunk = (sequence, KV head, row tile of 16 * NQ query rows,
// prefix split of up to pages_per_split pages). Blocks of up to 32 query rows
// run one single-wave workgroup per chunk; larger (GQA) blocks run the 2 or 4
// row tiles of a split as the waves of one workgroup that share one LDS ring,
// so a tile is loaded once per split rather than once per row tile. Split 0
// of every (sequence, head, row tile) also carries the draft block, in place
// of one prefix page, so every split streams the same number of tiles. The grid
// holds every chunk the block table's width allows; a chunk past its
// sequence's prefix exits at once, and the hardware dispatcher keeps the
// compute units fed as chunks finish. Workgroups are dealt to the 8 XCDs
// round-robin, so chunk c runs on XCD c mod 8; inside each run of 8 splits
// the row tiles of one split are numbered 8 apart, which puts them on one
// XCD, where they share its L2.
//
// A chunk fetches its sequence's prefix length, its page ids and its Q rows
// (into registers) in one memory round trip, then streams its 32-token tiles (two per prefix
// page, then the draft block's) through a ring of NB LDS slots filled by the
// direct-to-LDS loads of gfx950 (buffer_load_dwordx4 ... lds for prefix
// pages, global_load_lds_dwordx4 for the draft block), NB tiles ahead of the
// tile being computed; the loads of the next tile are spread over the
// computation of the current one. The wave waits on its own vector-memory
// counter for the data it reads. A prefix tile's loads address a buffer
// resource per page half with one per-lane offset and a uniform fragment
// offset in an SGPR.
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
// A chunk ends by writing its piece record (m, l and O / l in fp16 under a
// per-row power-of-two scale) to the workspace for the combine kernel, or,
// when its sequence has a single split, the normalised output. Query rows of a row tile: row = i * G + g (block position i,
// head kvh * G + g). Logits are scaled into base-2 units after the product,
// inside the exponent's fused multiply-add.

#include "mfma_tile.h"

namespace das {
namespace {

// Issue priority of a long chunk from the tiles it has left: among the
// chunks resident on a CU, the one with more work left issues first, so the
// long chunks of a ragged batch do not run alone at the end of the launch.
// Short chunks keep the hardware's oldest-first order, which measured better
// when the chunks are of equal length.
constexpr int kLongChunkTiles = 40;
__device__ __forceinline__ void prio_by_remaining(int rem) {
  if (rem > 24) __builtin_amdgcn_s_setprio(3);
  else if (rem > 12) __builtin_amdgcn_s_setprio(2);
  else if (rem > 4) __builtin_amdgcn_s_setprio(1);
  else __builtin_amdgcn_s_setprio(0);
}

// At least two waves per SIMD: the kernel then fits in 256 registers, so the
// output and score accumulators stay in VGPRs (the MFMAs write them there)
// instead of being copied out of AGPRs on every tile.
// NW = 1: one wave per chunk, its own ring. NW > 1: the NW row tiles of a
// split share one workgroup and one ring; each wave loads its own block of
// NF / NW consecutive fragments of a tile (whole 128-byte lines of the
// page), and one barrier per tile both publishes the tile and frees the slot
// read in the previous iteration, which is then refilled (NB - 1 tiles in
// flight).
template <int DH, int NQ, int NB, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2)))
void attn_mfma_kernel(AttnParams p, int n_rg, int n_chunks) {
  using G = Geo<DH, NQ, NB>;
  constexpr int KS = G::KS;
  constexpr int DT = G::DT;
  constexpr int NF = G::NF;
  constexpr int ROWS = 16 * NQ;
  __shared__ __attribute__((aligned(16))) uint8_t ring[NB * G::SLOT];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar branches
  const int ln = lane & 15;
  const int lg = lane >> 4;
  const int pps = p.pages_per_split;

  // chunk number -> (split group, row-tile group of NW row tiles): in each
  // complete run of 8 groups, row-tile group rg of group 8k + x is number
  // 8 n_rg k + 8 rg + x;
  // group = (split * B + b) * hkv + kvh, so every sequence's first split is
  // dispatched before any second split (the longest chunks first: a ragged
  // batch's short tails come last)
  int grp, rg;
  {
    const int c = blockIdx.x, span = 8 * n_rg, runs = (n_chunks / n_rg) >> 3;
    if (c < runs * span) {
      grp = 8 * (c / span) + (c % span & 7);
      rg = (c % span) >> 3;
    } else {
      grp = c / n_rg;
      rg = c % n_rg;
    }
  }
  const int rt = rg * NW + wave;  // this wave's row tile
  const int kvh = grp % p.hkv;
  const int b = (grp / p.hkv) % p.batch;
  const int split = grp / p.hkv / p.batch;
  const int pg0 = split_first_page(split, pps);
  const int pg_cap = split_first_page(split + 1, pps) - pg0;  // pages of a full split

  // one round trip: the prefix length, this split's page ids, the Q
  // fragments (B operand of S^T = K Q^T: lane holds dims 8g..8g+7 of row n,
  // loaded straight into registers)
  const int s_raw = p.prefix_len[b];
  int page_id = 0;  // lane i: page id of the split's i-th page
  if (lane < pg_cap && pg0 + lane < p.max_pages)
    page_id = p.block_table[static_cast<size_t>(b) * p.max_pages + pg0 + lane];
  u32x4 qf[NQ][KS];
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    // rows past the last are clamped; their outputs are never written
    const int row = min(rt * ROWS + qt * 16 + ln, p.rows - 1);
    const int i = row / p.group, g = row % p.group;
    const bf16_t *qrow = static_cast<const bf16_t *>(p.q) +
                         ((static_cast<size_t>(b) * p.w + i) * p.hq + kvh * p.group + g) * DH;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[qt][ks] = *reinterpret_cast<const u32x4 *>(qrow + 32 * ks + 8 * lg);
  }
  bool bad;
  const int S = clamp_prefix(s_raw, p.max_pages, &bad);
  if (bad && split == 0 && kvh == 0 && rt == 0 && lane == 0)
    report_error(p.dev_error, DAS_DEVERR_PREFIX);
  const int npages = (S + kPage - 1) / kPage;
  const int nsb = splits_of(npages, pps);  // splits of this sequence
  if (split >= nsb) return;
  // The round trip's loads (prefix length, page ids, Q fragments) are done
  // before any tile load is issued: the page ids are needed at once, and with
  // no load into registers left pending, the loop's waits count tile loads
  // only (otherwise a use of those registers inside the loop has to wait for
  // every load issued before it, prefetched tiles included).
  wait_vmcnt<0>();
  const int npg = max(0, min(pg_cap, npages - pg0));
  const int npg2 = 2 * npg;                                   // prefix tiles
  const int ntile = npg2 + (split == 0 ? (p.w + 31) >> 5 : 0);  // + draft-block tiles

  const char *kl = static_cast<const char *>(p.k_layer);
  const char *vl = static_cast<const char *>(p.v_layer);
  const size_t head_off = static_cast<size_t>(kvh) * p.num_pages * kPage * DH * 2;
  const size_t tok_bytes = static_cast<size_t>(p.hkv) * DH * 2;  // block row stride
  const char *kblk = static_cast<const char *>(p.kb) +
                     (static_cast<size_t>(b) * p.w * p.hkv + kvh) * DH * 2;
  const char *vblk = static_cast<const char *>(p.vb) +
                     (static_cast<size_t>(b) * p.w * p.hkv + kvh) * DH * 2;
  // per-lane byte offsets of the fragments inside a page: key token slot
  // 8(n/4) + n%4 (plus a uniform part), column 8g; value token group g of
  // the tile, head dim n
  const uint32_t lane_k = ((8 * (ln >> 2) + (ln & 3)) * DH + 8 * lg) * 2;
  const uint32_t lane_v = (lg * DH + ln) * 16;

  // Source of prefix tile t: its page's 32-token key half ([32][DH], at
  // kbase) and value half (token groups 4u .. 4u + 3 of [8][DH][8], at vbase),
  // resolved once per tile. An out-of-range page id is reported and read as
  // page 0 (its tile is masked out).
  auto tile_src = [&](int t, const char *&kbase, const char *&vbase) {
    const int page = __builtin_amdgcn_readlane(page_id, t >> 1);
    const bool ok = page >= 0 && page < p.num_pages;
    if (!ok) report_error(p.dev_error, DAS_DEVERR_PAGE);
    const size_t off = head_off + static_cast<size_t>(ok ? page : 0) * kPage * DH * 2;
    const int u = t & 1;
    kbase = kl + off + (32 * u) * DH * 2;
    vbase = vl + off + 64 * DH * u;
  };
  // fragment f of a tile is loaded by wave f / (NF / NW): a wave's fragments
  // cover whole 128-byte lines (the key fragments of one S^T half are the
  // 64-byte pieces of the same token rows), so no line is requested by two
  // waves
  auto mine = [&](int f) { return NW == 1 || f / (NF / NW) == wave; };
  // Loads of tile t into ring slot t % NB, in three parts (key fragments of
  // each S^T half, then the values) so they can be spread over the
  // computation of the previous tile. Both halves span 64 * DH bytes.
  auto issue_part = [&](int t, int part, const char *kbase, const char *vbase) {
    uint8_t *slot = ring + (t % NB) * G::SLOT;
    if (t < npg2) {
      if (part < 2) {
        const auto r = buffer_of(kbase, 64 * DH);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          if (mine(part * KS + ks))
            dma16(r, lane_k, (4 * part * DH + 32 * ks) * 2, slot + (part * KS + ks) * kFragBytes);
      } else {
        const auto r = buffer_of(vbase, 64 * DH);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          if (mine(2 * KS + dt)) dma16(r, lane_v, 256 * dt, slot + (2 * KS + dt) * kFragBytes);
      }
    } else {
      // draft block tile u: key fragments by token slot, value rows raw
      const int u = t - npg2;
      if (part < 2) {
        const int tok = min(32 * u + 8 * (ln >> 2) + 4 * part + (ln & 3), p.w - 1);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          if (mine(part * KS + ks))
            dma16(kblk + tok * tok_bytes + (32 * ks + 8 * lg) * 2, slot + (part * KS + ks) * kFragBytes);
      } else {
#pragma unroll
        for (int f = 0; f < DT; ++f) {
          if (!mine(2 * KS + f)) continue;
          const int o = f * kFragBytes + 16 * lane;  // byte in the [32][DH] half
          const int tok = min(32 * u + o / (2 * DH), p.w - 1);
          dma16(vblk + tok * tok_bytes + o % (2 * DH), slot + (2 * KS + f) * kFragBytes);
        }
      }
    }
  };

  // A shared-ring wave's loads of prefix tile t: its own block of NF / NW
  // fragments, which is whole key halves or whole value groups, so the
  // fragment offsets are scalars and no per-fragment test is made.
  auto issue_own_prefix = [&](int t, const char *kbase, const char *vbase) {
    constexpr int FPW = NF / NW;
    static_assert(NW == 1 || (2 * KS) % FPW == 0, "a wave loads keys only or values only");
    uint8_t *slot = ring + (t % NB) * G::SLOT;
    const int f0 = wave * FPW;
    if (f0 < 2 * KS) {
      const auto r = buffer_of(kbase, 64 * DH);
#pragma unroll
      for (int i = 0; i < FPW; ++i) {
        const int f = f0 + i, part = f / KS, ks = f - part * KS;
        dma16(r, lane_k, (4 * part * DH + 32 * ks) * 2, slot + f * kFragBytes);
      }
    } else {
      const auto r = buffer_of(vbase, 64 * DH);
#pragma unroll
      for (int i = 0; i < FPW; ++i) {
        const int dt = f0 - 2 * KS + i;
        dma16(r, lane_v, 256 * dt, slot + (2 * KS + dt) * kFragBytes);
      }
    }
  };

  int n_issued = 0;
  for (; n_issued < NB && n_issued < ntile; ++n_issued) {
    const char *kbase = kl, *vbase = vl;
    if (n_issued < npg2) tile_src(n_issued, kbase, vbase);
    for (int part = 0; part < 3; ++part) issue_part(n_issued, part, kbase, vbase);
  }

  int cap_blk[NQ];
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) cap_blk[qt] = (rt * ROWS + qt * 16 + ln) / p.group;  // block position i
  State<DH, NQ> st;
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    st.m[qt] = kNegInf;
    st.l[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) st.o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Tile t's fragments from its ring slot into registers (keys; values as
  // V^T fragments, the draft block's token-major values gathered), and which
  // of its tokens each row sees.
  auto read_tile = [&](int t, u32x4 (&kf)[2][KS], u32x4 (&vf)[DT], int (&cap)[NQ], int &limit,
                       bool &full) {
    const uint8_t *slot = ring + (t % NB) * G::SLOT;
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kf[e][ks] = *reinterpret_cast<const u32x4 *>(slot + (e * KS + ks) * kFragBytes + 16 * lane);
    if (t < npg2) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        vf[dt] = *reinterpret_cast<const u32x4 *>(slot + (2 * KS + dt) * kFragBytes + 16 * lane);
      const int page = __builtin_amdgcn_readlane(page_id, t >> 1);
      const bool ok = page >= 0 && page < p.num_pages;
      limit = ok ? min(32, S - (pg0 + (t >> 1)) * kPage - 32 * (t & 1)) : 0;
      full = limit >= 32;
      if (!full) {
        // Invisible tokens (past the prefix, or an unreadable page) enter P.V
        // with probability 0; their values are zeroed so that whatever the
        // cache holds there (NaN, Inf) contributes nothing. Lane group lg
        // holds tokens 8 lg .. 8 lg + 7 of the tile, two per 32-bit word.
        const int nv = min(max(limit - 8 * lg, 0), 8);
        u32x4 keep;
#pragma unroll
        for (int k = 0; k < 4; ++k)
          keep[k] = (2 * k < nv ? 0xffffu : 0u) | (2 * k + 1 < nv ? 0xffff0000u : 0u);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) vf[dt] &= keep;
      }
#pragma unroll
      for (int qt = 0; qt < NQ; ++qt) cap[qt] = 0x7fffffff;
    } else {
      // block values are token-major [32][DH] in the slot: gather V^T
      const int u = t - npg2;
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
  };

  if constexpr (NW == 1) {
  const bool long_chunk = ntile > kLongChunkTiles;
  for (int t = 0; t < ntile; ++t) {
    if (long_chunk) prio_by_remaining(ntile - t);
    wait_tiles<NF>(n_issued - t - 1);
    u32x4 kf[2][KS], vf[DT];
    int cap[NQ];
    int limit;
    bool full;
    read_tile(t, kf, vf, cap, limit, full);
    // the slot's fragments are in registers before it is refilled
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)
    const int next = n_issued;
    const bool refill = next < ntile;
    if (refill) ++n_issued;
    const char *kbase = kl, *vbase = vl;
    if (refill && next < npg2) tile_src(next, kbase, vbase);
    compute_tile<DH, NQ, true>(st, kf, vf, qf, cap, limit, full, p.scale_log2, lg, [&](int part) {
      if (refill) issue_part(next, part, kbase, vbase);
    });
  }

  } else {
  for (int t = 0; t < ntile; ++t) {
    wait_tiles<NF / NW>(n_issued - t - 1);  // this wave's loads of tile t have landed
    // every wave's loads of tile t have landed, and every wave has read slot
    // (t - 1) % NB, which now takes tile t - 1 + NB
    __syncthreads();
    if (t >= 1 && n_issued < ntile) {
      const char *kbase = kl, *vbase = vl;
      if (n_issued < npg2) {
        tile_src(n_issued, kbase, vbase);
        issue_own_prefix(n_issued, kbase, vbase);
      } else {
        for (int part = 0; part < 3; ++part) issue_part(n_issued, part, kbase, vbase);
      }
      ++n_issued;
    }
    u32x4 kf[2][KS], vf[DT];
    int cap[NQ];
    int limit;
    bool full;
    read_tile(t, kf, vf, cap, limit, full);
    // the slot's fragments are in registers before the next barrier
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)
    compute_tile<DH, NQ, true>(st, kf, vf, qf, cap, limit, full, p.scale_log2, lg, [](int) {});
  }

  }

  // Chunk result. Lane holds head dims 16dt + 4g .. +3 of row n of tile qt.
  uint8_t *prec = reinterpret_cast<uint8_t *>(p.ws_o) +
                  ((static_cast<size_t>(b) * p.hkv + kvh) * p.nsplit + split) * p.piece_stride;
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) {
    const int row = rt * ROWS + qt * 16 + ln;
    if (row >= p.rows) continue;
    const float lrow = group_sum(st.l[qt]);  // row sum from its 4 lanes, all live
    if (nsb == 1) {
      const float inv = 1.f / lrow;
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
            (st.m[qt] + log2f(lrow)) * 0.69314718055994530942f;
    } else {
      write_piece_row<DH>(prec, p.rows, row, lg, st.o[qt], st.m[qt], lrow);
    }
  }
}

template <int DH, int NQ, int NB, int NW>
hipError_t launch_typed(const AttnParams &p, hipStream_t s) {
  const int n_rt = (p.rows + 16 * NQ - 1) / (16 * NQ);
  const int n_rg = (n_rt + NW - 1) / NW;  // row-tile groups (workgroups) per split
  // every possible chunk (the table width bounds the splits of a sequence)
  const long chunks = static_cast<long>(p.batch) * p.hkv * p.nsplit * n_rg;
  if (chunks > 0x7fffffffL) return hipErrorInvalidValue;
  return launch_kernel(attn_mfma_kernel<DH, NQ, NB, NW>, dim3(static_cast<unsigned>(chunks)),
                       dim3(64 * NW), s, p, n_rg, static_cast<int>(chunks));
}

// Up to 32 query rows: one wave per chunk. More rows (GQA blocks): the row
// tiles of a split share a workgroup and one ring, so each tile enters LDS
// once per split instead of once per row tile. Four row tiles and more: four
// waves and a 4-deep ring (two workgroups per CU; long-prefix GQA 0.33 ->
// 0.41 of HBM peak); two row tiles: two waves and a 2-deep ring (a 4-deep
// one would leave one wave per SIMD at head dim 128).
template <int DH>
hipError_t launch_dh(const AttnParams &p, hipStream_t s) {
  static_assert(mfma_tiles_per_wave(16) == 1 && mfma_tiles_per_wave(17) == 2 &&
                mfma_waves(32) == 1 && mfma_waves(64) == 2 && mfma_waves(65) == 4,
                "host-side grid checks mirror these shapes");
  if (p.rows <= 16) return launch_typed<DH, 1, 2, 1>(p, s);
  if (p.rows <= 32) return launch_typed<DH, 2, 2, 1>(p, s);
  if (p.rows <= 64) return launch_typed<DH, 2, 2, 2>(p, s);
  return launch_typed<DH, 2, 4, 4>(p, s);
}

}  // namespace

hipError_t launch_attn_mfma(const AttnParams &p, int dh, hipStream_t s) {
  if (dh == 64) return launch_dh<64>(p, s);
  if (dh == 96) return launch_dh<96>(p, s);
  return launch_dh<128>(p, s);
}

}  // namespace das
