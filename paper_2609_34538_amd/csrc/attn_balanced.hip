// Balanced persistent matrix-core attention for batches of sequences with
// different prefix lengths (Eq. (2)-(3) over a ragged batch).
//
// Work layout. A unit is one (sequence b, KV head) pair: its query block
// (w * G <= 32 rows) against the sequence's prefix and the draft block. A
// unit has 2 * ceil(S_b / 64) prefix tiles of 32 tokens (two per page) and
// ceil(w / 32) block tiles, in that order. The units of all sequences, laid
// end to end (sequence-major, then KV head), form one global sequence of T
// tiles. Worker j of W (single-wave workgroups, balanced_workers_per_cu of
// them per compute unit, all resident at once) takes the tiles
// [T j / W, T (j + 1) / W): every worker streams
// the same number of tiles (+-1), whatever the lengths, so the launch has no
// tail of long chunks and no idle slots while short ones finish.
//
// A worker streams its tiles through a two-slot LDS ring (the direct-to-LDS
// loads of the split-grid kernel) without pausing at unit boundaries: while
// tile k is computed, tile k + 1 is loaded into the other slot. Page ids come
// from a 64-entry window in registers; the unit's next window, the next
// unit's first window and (one row tile per wave) the next unit's Q rows are
// loaded a window or a unit ahead. One tile in flight per wave: on the
// batched workloads this measured faster than keeping two tiles in flight
// (the split-grid kernel's depth), 0.72-0.73 against 0.68-0.69 of 8 TB/s on
// the same box. At the end
// of a unit (or of its range) the worker writes the unit's normalised output
// when it processed the whole unit, otherwise a piece (the running maximum
// m, the sum l and the normalised output O / l in fp16 under a per-row
// power-of-two scale) that the merge kernel combines with the unit's other
// pieces. Only the range's first unit can end as a piece in the middle of
// the range; its record waits in LDS and is written with the range's last
// flush, because writes in the middle of the stream delay the reads at the
// DRAM (width-32 calls 0.768 -> 0.788 and 0.771 -> 0.805 of 8 TB/s, ragged
// batch 0.702 -> 0.720, same process).
// Pieces are indexed unit + worker: along the tile sequence either the unit
// or the worker (or both) advances, so the index is unique, and a unit's
// pieces are consecutive.
//
// Both the attention kernel and the merge derive T, W and every unit's tile
// range from the prefix lengths on the device (one length per lane, a wave
// prefix sum), so the host needs no synchronisation. Batches of at most 64
// sequences.

#include "mfma_tile.h"

namespace das {
namespace {

constexpr int kMinTilesPerWorker = 16;  // fewer tiles per worker: fewer workers

__device__ __forceinline__ long long readlane64(long long x, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(x), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(x >> 32), lane);
  return static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo);
}

// A wave-uniform pointer, held in scalar registers (the compiler cannot
// always prove the uniformity of values carried across the loop, and a
// buffer resource built from a vector register costs a waterfall loop).
__device__ __forceinline__ const char *uniform_ptr(const char *ptr) {
  const uint64_t v = reinterpret_cast<uint64_t>(ptr);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return reinterpret_cast<const char *>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Inclusive prefix sum over the wave's 64 lanes.
__device__ __forceinline__ long long wave_incl_scan(long long x, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const long long y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

// The tile numbering of one call, identical in the attention and the merge
// kernels: lane b < B holds sequence b's clamped prefix length, its tiles
// per unit and the inclusive prefix sum of the tiles of sequences 0..b.
struct TileMap {
  int s;            // lane b: prefix length S_b (clamped)
  int tu;           // lane b: tiles per unit of sequence b
  long long incl;   // lane b: tiles of the units of sequences 0..b
  long long total;  // T
  long long workers;  // W (wave-uniform)
};

__device__ __forceinline__ TileMap tile_map(const AttnParams &p, int lane, bool report) {
  TileMap m;
  const int s_raw = lane < p.batch ? p.prefix_len[lane] : 0;
  bool bad;
  m.s = clamp_prefix(s_raw, p.max_pages, &bad);
  if (report && bad && lane < p.batch) report_error(p.dev_error, DAS_DEVERR_PREFIX);
  m.tu = 2 * ((m.s + kPage - 1) / kPage) + ((p.w + 31) >> 5);
  const long long own = lane < p.batch ? static_cast<long long>(m.tu) * p.hkv : 0;
  m.incl = wave_incl_scan(own, lane);
  m.total = readlane64(m.incl, 63);
  long long w = m.total / kMinTilesPerWorker;
  if (w < 1) w = 1;
  m.workers = w < p.n_workers ? w : p.n_workers;
  return m;
}

// The worker whose range holds global tile g: the largest j with
// floor(T j / W) <= g.
__device__ __forceinline__ long long worker_of(long long g, long long T, long long W) {
  return ((g + 1) * W - 1) / T;
}

// Position of a worker in the tile sequence: unit (b, kvh), tile t of the
// unit, and the unit's shape. Wave-uniform.
struct Cursor {
  int b, kvh, t;
  int s, np, tu;  // prefix length, prefix pages, tiles of the unit
};

// The same cursor, pinned to scalar registers: values carried around the
// tile loop are otherwise taken for divergent and kept (and branched on) in
// vector registers.
__device__ __forceinline__ Cursor uniform(const Cursor &x) {
  Cursor y;
  y.b = __builtin_amdgcn_readfirstlane(x.b);
  y.kvh = __builtin_amdgcn_readfirstlane(x.kvh);
  y.t = __builtin_amdgcn_readfirstlane(x.t);
  y.s = __builtin_amdgcn_readfirstlane(x.s);
  y.np = __builtin_amdgcn_readfirstlane(x.np);
  y.tu = __builtin_amdgcn_readfirstlane(x.tu);
  return y;
}

template <int DH, int NQ>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2)))
void attn_balanced_kernel(AttnParams p) {
  using G = Geo<DH, NQ, 2>;
  constexpr int KS = G::KS;
  constexpr int DT = G::DT;
  __shared__ __attribute__((aligned(16))) uint8_t ring[2 * G::SLOT];
  // the record of a piece that ends in the middle of the range (only the
  // range's first unit can), written to global memory with the range's last
  // flush
  constexpr int kStash = static_cast<int>(piece_record_bytes(balanced_max_rows(DH), DH));
  __shared__ __attribute__((aligned(16))) uint8_t stash[kStash];
  static_assert(2 * G::SLOT + kStash == balanced_lds_per_worker(DH),
                "the host's worker count assumes this LDS per worker");

  const int lane = threadIdx.x;
  const int ln = lane & 15;
  const int lg = lane >> 4;
  const int j = blockIdx.x;

  const TileMap tm = tile_map(p, lane, j == 0);
  if (j >= tm.workers) return;
  const long long T = tm.total, W = tm.workers;
  const long long g0 = T * j / W;
  const long long n = T * (j + 1) / W - g0;  // >= 1: W <= max(1, T / 16)

  // the unit holding g0: sequences ending at or before g0 come first
  const uint64_t done = __builtin_amdgcn_ballot_w64(lane < p.batch && tm.incl <= g0);
  Cursor c0;
  c0.b = __builtin_amdgcn_readfirstlane(__builtin_popcountll(done));
  c0.s = __builtin_amdgcn_readlane(tm.s, c0.b);
  c0.np = (c0.s + kPage - 1) / kPage;
  c0.tu = __builtin_amdgcn_readlane(tm.tu, c0.b);
  {
    const long long seq_start = readlane64(tm.incl, c0.b) -
                                static_cast<long long>(c0.tu) * p.hkv;
    const long long local = g0 - seq_start;
    c0.kvh = static_cast<int>(local / c0.tu);
    c0.t = static_cast<int>(local % c0.tu);
  }
  const char *kl = static_cast<const char *>(p.k_layer);
  const char *vl = static_cast<const char *>(p.v_layer);
  const size_t tok_bytes = static_cast<size_t>(p.hkv) * DH * 2;  // block row stride
  // per-lane byte offsets of a fragment inside a page half (as in the
  // split-grid kernel): key token slot 8(n/4) + n%4, column 8g; value token
  // group g, head dim n
  const uint32_t lane_k = ((8 * (ln >> 2) + (ln & 3)) * DH + 8 * lg) * 2;
  const uint32_t lane_v = (lg * DH + ln) * 16;

  // Q fragments of a unit (B operand of S^T = K Q^T: lane holds dims
  // 8g..8g+7 of row n); rows past the block's last are clamped and never
  // written
  auto q_row = [&](const Cursor &x, int qt) {
    const int row = min(qt * 16 + ln, p.rows - 1);
    const int i = row / p.group, g = row % p.group;
    return static_cast<const bf16_t *>(p.q) +
           ((static_cast<size_t>(x.b) * p.w + i) * p.hq + x.kvh * p.group + g) * DH;
  };
  auto load_q = [&](const Cursor &x, u32x4 (&qf)[NQ][KS]) {
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      const int row = min(qt * 16 + ln, p.rows - 1);
      const int i = row / p.group, g = row % p.group;
      const bf16_t *qrow = static_cast<const bf16_t *>(p.q) +
                           ((static_cast<size_t>(x.b) * p.w + i) * p.hq + x.kvh * p.group + g) * DH;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[qt][ks] = *reinterpret_cast<const u32x4 *>(qrow + 32 * ks + 8 * lg);
    }
  };
  // Sources of a tile: a prefix tile's 32-token key half and value half of
  // its page; an out-of-range page id is reported and read as page 0 (the
  // tile is then masked out).
  auto tile_src = [&](const Cursor &x, int page, const char *&kbase, const char *&vbase,
                      bool &ok) {
    kbase = kl;
    vbase = vl;
    ok = true;
    if (x.t >= 2 * x.np) return;
    ok = page >= 0 && page < p.num_pages;
    if (!ok) report_error(p.dev_error, DAS_DEVERR_PAGE);
    const size_t off = (static_cast<size_t>(x.kvh) * p.num_pages + (ok ? page : 0)) *
                       kPage * DH * 2;
    const int u = x.t & 1;
    kbase = kl + off + (32 * u) * DH * 2;
    vbase = vl + off + 64 * DH * u;
  };
  // Loads of a tile into ring slot `si`, in three parts (key fragments of
  // each S^T half, then the values) spread over the computation of the
  // previous tile.
  auto issue_part = [&](int si, const Cursor &x, int part, const char *kbase,
                        const char *vbase) {
    uint8_t *slot = ring + si * G::SLOT;
    if (x.t < 2 * x.np) {
      if (part < 2) {
        const auto r = buffer_of(uniform_ptr(kbase), 64 * DH);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          dma16(r, lane_k, (4 * part * DH + 32 * ks) * 2, slot + (part * KS + ks) * kFragBytes);
      } else {
        const auto r = buffer_of(uniform_ptr(vbase), 64 * DH);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          dma16(r, lane_v, 256 * dt, slot + (2 * KS + dt) * kFragBytes);
      }
    } else {
      // draft block tile u: key fragments by token slot, value rows raw
      const int u = x.t - 2 * x.np;
      const size_t row0 = static_cast<size_t>(x.b) * p.w * p.hkv + x.kvh;
      const char *kblk = static_cast<const char *>(p.kb) + row0 * DH * 2;
      const char *vblk = static_cast<const char *>(p.vb) + row0 * DH * 2;
      if (part < 2) {
        const int tok = min(32 * u + 8 * (ln >> 2) + 4 * part + (ln & 3), p.w - 1);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          dma16(kblk + tok * tok_bytes + (32 * ks + 8 * lg) * 2,
                slot + (part * KS + ks) * kFragBytes);
      } else {
#pragma unroll
        for (int f = 0; f < DT; ++f) {
          const int o = f * kFragBytes + 16 * lane;  // byte in the [32][DH] half
          const int tok = min(32 * u + o / (2 * DH), p.w - 1);
          dma16(vblk + tok * tok_bytes + o % (2 * DH), slot + (2 * KS + f) * kFragBytes);
        }
      }
    }
  };

  State<DH, NQ> st;
  auto reset = [&]() {
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      st.m[qt] = kNegInf;
      st.l[qt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) st.o[qt][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  // End of a unit's stretch in this worker: the normalised output when the
  // worker processed the whole unit, else a piece for the merge. Lane holds
  // head dims 16dt + 4g .. +3 of row n of tile qt.
  auto flush = [&](const Cursor &x, bool whole, uint8_t *rec) {
#pragma unroll
    for (int qt = 0; qt < NQ; ++qt) {
      const int row = qt * 16 + ln;
      if (row >= p.rows) continue;
      if (whole) {
        const float inv = 1.f / st.l[qt];
        const int i = row / p.group, h = x.kvh * p.group + row % p.group;
        bf16_t *orow = static_cast<bf16_t *>(p.out) +
                       ((static_cast<size_t>(x.b) * p.w + i) * p.hq + h) * DH;
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
          p.lse[(static_cast<size_t>(x.b) * p.hq + h) * p.w + i] =
              (st.m[qt] + log2f(st.l[qt])) * 0.69314718055994530942f;
      } else {
        // a piece record of its own (256-byte aligned, so its lines are
        // written by this wave alone), in half the bytes of fp32 partials:
        // the stores of a piece written in the middle of a worker's range
        // delay its next tile waits
        write_piece_row<DH>(rec, p.rows, row, lg, st.o[qt], st.m[qt], st.l[qt]);
      }
    }
  };

  // block position of each row (the causal cap on the block tiles)
  int cap_blk[NQ];
#pragma unroll
  for (int qt = 0; qt < NQ; ++qt) cap_blk[qt] = (qt * 16 + ln) / p.group;

  // Page ids of the sequence of the current unit, 64 at a time: lane i holds
  // the id of page pw0 + i (0 past the table's width).
  auto load_window = [&](int b, int pw0) -> int {
    const int pg = pw0 + lane;
    return pg < p.max_pages ? p.block_table[static_cast<size_t>(b) * p.max_pages + pg] : 0;
  };
  auto next_unit = [&](const Cursor &x) {
    Cursor y = x;
    y.t = 0;
    if (++y.kvh == p.hkv) {
      y.kvh = 0;
      ++y.b;
      y.s = __builtin_amdgcn_readlane(tm.s, y.b);
      y.np = (y.s + kPage - 1) / kPage;
      y.tu = __builtin_amdgcn_readlane(tm.tu, y.b);
    }
    return uniform(y);
  };

  // Outer loop: the units of this worker's range; inner loop: the unit's
  // tiles in the range, tile t computed while tile t + 1 (or the next unit's
  // first tile) is loaded into the other ring slot. The next unit's Q rows
  // and first page window, and the current unit's next page window, are
  // loaded one window or one unit ahead; the wait at the top of every tile
  // completes them with the tile.
  Cursor cu = c0;
  int pw0 = (c0.t >> 1) & ~63;
  int pwin = load_window(cu.b, pw0);
  int x_pw0 = -1;  // first page of the prefetched next window (-1: none)
  int pwin_x = 0;
  if (pw0 + 64 < cu.np) {
    x_pw0 = pw0 + 64;
    pwin_x = load_window(cu.b, x_pw0);
  }
  // With one row tile per wave the next unit's Q rows are loaded at the
  // start of the current unit (qn); with two there is no room for a second
  // set, and they are loaded when the unit starts (one round trip per unit).
  constexpr bool kPrefetchQ = NQ == 1;
  u32x4 qf[NQ][KS], qn[kPrefetchQ ? NQ : 1][KS];
  load_q(cu, qf);
  wait_vmcnt<0>();
  const char *kbase, *vbase;
  bool ok_cur;
  {
    const int pg = cu.t >> 1;
    tile_src(cu, __builtin_amdgcn_readlane(pwin, pg - pw0), kbase, vbase, ok_cur);
    for (int part = 0; part < 3; ++part) issue_part(0, cu, part, kbase, vbase);
  }
  long long g_unit = g0 - c0.t;  // global index of the current unit's first tile
  uint8_t *stash_dst = nullptr;  // global record of the stashed piece
  int si = 0;                // ring slot of the tile being computed
  long long remaining = n;   // tiles left in this worker's range
  for (;;) {
    const int t_first = cu.t;
    const int t_end = static_cast<int>(min(static_cast<long long>(cu.tu), t_first + remaining));
    const bool has_next = remaining > t_end - t_first;
    Cursor nu = cu;
    int pwin_n = 0;
    if (has_next) {
      nu = next_unit(cu);
      pwin_n = load_window(nu.b, 0);
      if constexpr (kPrefetchQ) {
        const bf16_t *qrow = q_row(nu, 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          qn[0][ks] = *reinterpret_cast<const u32x4 *>(qrow + 32 * ks + 8 * lg);
      }
    }
    reset();
    for (int t = t_first; t < t_end; ++t) {
      wait_vmcnt<0>();  // tile t, and every window and Q load issued before it
      const uint8_t *slot = ring + si * G::SLOT;
      u32x4 kf[2][KS], vf[DT];
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          kf[e][ks] = *reinterpret_cast<const u32x4 *>(slot + (e * KS + ks) * kFragBytes + 16 * lane);
      const bool prefix_tile = t < 2 * cu.np;
      int cap[NQ];
      int limit;
      bool full;
      if (prefix_tile) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          vf[dt] = *reinterpret_cast<const u32x4 *>(slot + (2 * KS + dt) * kFragBytes + 16 * lane);
        limit = ok_cur ? min(32, cu.s - 32 * t) : 0;
        full = limit >= 32;
        if (!full) {
          // invisible tokens enter P.V with probability 0; their values are
          // zeroed so whatever the page holds there (NaN, Inf) adds nothing
          const int nv = min(max(limit - 8 * lg, 0), 8);
          u32x4 keep;
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4)
            keep[q4] = (2 * q4 < nv ? 0xffffu : 0u) | (2 * q4 + 1 < nv ? 0xffff0000u : 0u);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) vf[dt] &= keep;
        }
#pragma unroll
        for (int qt = 0; qt < NQ; ++qt) cap[qt] = 0x7fffffff;
      } else {
        // block values are token-major [32][DH] in the slot: gather V^T
        const int ub = t - 2 * cu.np;
        const uint16_t *raw = reinterpret_cast<const uint16_t *>(slot + 2 * KS * kFragBytes);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          u16x8 v8;
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) v8[jj] = raw[(8 * lg + jj) * DH + 16 * dt + ln];
          vf[dt] = __builtin_bit_cast(u32x4, v8);
        }
        limit = p.w - 32 * ub;
        full = false;
#pragma unroll
        for (int qt = 0; qt < NQ; ++qt) cap[qt] = cap_blk[qt] - 32 * ub;
      }
      // the slot's fragments are in registers before the other slot is
      // refilled, and the refill below completes the previous reads
      __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)

      // the next tile: this unit's t + 1, or the next unit's first tile
      const bool in_unit = t + 1 < t_end;
      const bool refill = in_unit || has_next;
      Cursor ci = in_unit ? cu : nu;
      ci.t = in_unit ? t + 1 : 0;
      ci = uniform(ci);
      if (refill) {
        int page = 0;
        if (ci.t < 2 * ci.np) {
          const int pg = ci.t >> 1;
          if (!in_unit) {
            page = __builtin_amdgcn_readlane(pwin_n, pg);
          } else {
            if (pg - pw0 >= 64) {  // the next window of this unit
              pwin = pwin_x;
              pw0 = x_pw0;
              x_pw0 = -1;
            }
            page = __builtin_amdgcn_readlane(pwin, pg - pw0);
            // first issue in a window: load the one after it
            if (x_pw0 < 0 && pw0 + 64 < cu.np) {
              x_pw0 = pw0 + 64;
              pwin_x = load_window(cu.b, x_pw0);
            }
          }
        }
        tile_src(ci, page, kbase, vbase, ok_cur);  // ok_cur now describes tile t + 1
      }
      const int sn = si ^ 1;
      compute_tile<DH, NQ>(st, kf, vf, qf, cap, limit, full, p.scale_log2, lg, [&](int part) {
        if (refill) issue_part(sn, ci, part, kbase, vbase);
      });
      si = sn;
    }
    {
      const bool whole = t_first == 0 && t_end == cu.tu;
      const bool last = remaining <= t_end - t_first;
      const size_t piece = static_cast<size_t>(cu.b) * p.hkv + cu.kvh + j;
      uint8_t *grec = reinterpret_cast<uint8_t *>(p.ws_o) + piece * p.piece_stride;
      if (!whole && !last && stash_dst == nullptr) {
        flush(cu, false, stash);
        stash_dst = grec;
      } else {
        flush(cu, whole, grec);
      }
    }
    if (t_first == 0 && lane == 0) {
      // this worker holds the unit's first tile: record where the unit's
      // pieces start and how many workers share it, for the merge
      const long long jl = worker_of(g_unit + cu.tu - 1, T, W);
      const int unit = cu.b * p.hkv + cu.kvh;
      p.ws_rec[2 * unit] = unit + j;
      p.ws_rec[2 * unit + 1] = static_cast<int>(jl - j + 1);
    }
    g_unit += cu.tu;
    remaining -= t_end - t_first;
    if (remaining <= 0) {
      if (stash_dst) {
        const int bytes = p.rows * (DH * 2 + 16);
        for (int off = 16 * lane; off < bytes; off += 1024)
          *reinterpret_cast<u32x4 *>(stash_dst + off) = *reinterpret_cast<const u32x4 *>(stash + off);
      }
      break;
    }
    cu = nu;
    pwin = pwin_n;
    pw0 = 0;
    x_pw0 = -1;
    if constexpr (kPrefetchQ) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[0][ks] = qn[0][ks];
    } else {
      load_q(cu, qf);
    }
  }
}

// Merge of a unit's pieces (as the split-grid kernel's merge, over the pieces
// of the workers that share the unit): one 256-thread workgroup per unit,
// each thread holding IT (row, 4 columns) items and issuing the loads of all
// of them at once, so the merge costs two memory round trips (the record,
// then the pieces) whatever the block width, and a unit held whole by one
// worker occupies four waves for one round trip only. The unit's first piece
// and piece count come from the record its first worker wrote.
constexpr int kMergeThreads = 256;
constexpr int kEager = 4;  // pieces per item loaded at once (units rarely have more)

template <int DH>
constexpr int merge_items(int rows) {
  return (rows * (DH / 4) + kMergeThreads - 1) / kMergeThreads;
}
static_assert(merge_items<64>(32) == 2 && merge_items<96>(32) == 3 && merge_items<128>(16) == 2,
              "items per merge thread at the largest balanced blocks");

template <typename T, int DH, int IT>
__global__ __launch_bounds__(kMergeThreads) void attn_balanced_combine_kernel(AttnParams p) {
  const int unit = blockIdx.x;  // b * hkv + kvh
  const int piece0 = p.ws_rec[2 * unit];
  const int np = p.ws_rec[2 * unit + 1];
  if (np <= 1) return;  // written by its worker
  constexpr int CG = DH / 4;  // column groups of a row
  const int n_items = p.rows * CG;
  const int b = unit / p.hkv, kvh = unit % p.hkv;
  const size_t stride = static_cast<size_t>(p.piece_stride);
  const uint8_t *rec0 = reinterpret_cast<const uint8_t *>(p.ws_o) + piece0 * stride;
  const uint8_t *orow[IT], *mrow[IT];
  f32x4 meta[IT][kEager];
  h16x4 ov[IT][kEager];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    // items past the block's last repeat the first (computed, never stored)
    const int item0 = threadIdx.x + it * kMergeThreads;
    const int item = item0 < n_items ? item0 : 0;
    const int row = item / CG, c = 4 * (item % CG);
    orow[it] = rec0 + (row * DH + c) * 2;
    mrow[it] = rec0 + p.rows * DH * 2 + row * 16;
#pragma unroll
    for (int k = 0; k < kEager; ++k) {
      if (k < np) {  // uniform over the workgroup
        meta[it][k] = *reinterpret_cast<const f32x4 *>(mrow[it] + k * stride);
        ov[it][k] = *reinterpret_cast<const h16x4 *>(orow[it] + k * stride);
      }
    }
  }
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int item = threadIdx.x + it * kMergeThreads;
    // piece k: maximum meta[0], sum meta[1], unnormalised output = stored * meta[2]
    float mx = -__builtin_huge_valf();
#pragma unroll
    for (int k = 0; k < kEager; ++k) mx = k < np ? fmaxf(mx, meta[it][k][0]) : mx;
    float den = 0.f, n0 = 0.f, n1 = 0.f, n2 = 0.f, n3 = 0.f;
#pragma unroll
    for (int k = 0; k < kEager; ++k) {
      if (k < np) {
        const float sc = exp2f(meta[it][k][0] - mx);
        const float w = sc * meta[it][k][2];
        den += sc * meta[it][k][1];
        n0 += w * static_cast<float>(ov[it][k][0]);
        n1 += w * static_cast<float>(ov[it][k][1]);
        n2 += w * static_cast<float>(ov[it][k][2]);
        n3 += w * static_cast<float>(ov[it][k][3]);
      }
    }
    for (int k = kEager; k < np; ++k) {
      const f32x4 mk = *reinterpret_cast<const f32x4 *>(mrow[it] + k * stride);
      const h16x4 o = *reinterpret_cast<const h16x4 *>(orow[it] + k * stride);
      const float nm = fmaxf(mx, mk[0]);
      const float a = exp2f(mx - nm), sc = exp2f(mk[0] - nm);
      const float w = sc * mk[2];
      den = den * a + sc * mk[1];
      n0 = n0 * a + w * static_cast<float>(o[0]);
      n1 = n1 * a + w * static_cast<float>(o[1]);
      n2 = n2 * a + w * static_cast<float>(o[2]);
      n3 = n3 * a + w * static_cast<float>(o[3]);
      mx = nm;
    }
    if (item >= n_items) continue;
    const int row = item / CG, c = 4 * (item % CG);
    const int i = row / p.group, h = kvh * p.group + row % p.group;
    T *out = static_cast<T *>(p.out) + ((static_cast<size_t>(b) * p.w + i) * p.hq + h) * DH + c;
    const float inv = 1.f / den;
    out[0] = from_f32<T>(n0 * inv);
    out[1] = from_f32<T>(n1 * inv);
    out[2] = from_f32<T>(n2 * inv);
    out[3] = from_f32<T>(n3 * inv);
    if (p.lse && c == 0)
      p.lse[(static_cast<size_t>(b) * p.hq + h) * p.w + i] =
          (mx + log2f(den)) * 0.69314718055994530942f;
  }
}

// Blocks of up to 16 query rows: one row tile per wave; 17..32 rows: two
// (head dims 64 and 96 only: at 128 the second tile does not fit in the
// wave's registers, and such requests keep the split grid).
template <int DH>
hipError_t launch_dh(const AttnParams &p, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(p.n_workers));
  static_assert(balanced_max_rows(DH) == (DH == 128 ? 16 : 32), "launch shapes");
  if (p.rows <= 16) return launch_kernel(attn_balanced_kernel<DH, 1>, grid, dim3(64), s, p);
  if constexpr (DH == 128) return hipErrorInvalidValue;
  else return launch_kernel(attn_balanced_kernel<DH, 2>, grid, dim3(64), s, p);
}

template <int DH>
hipError_t launch_combine_dh(const AttnParams &p, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(p.batch * p.hkv)), block(kMergeThreads);
  switch (merge_items<DH>(p.rows)) {
    case 1: return launch_kernel(attn_balanced_combine_kernel<bf16_t, DH, 1>, grid, block, s, p);
    case 2: return launch_kernel(attn_balanced_combine_kernel<bf16_t, DH, 2>, grid, block, s, p);
    case 3: return launch_kernel(attn_balanced_combine_kernel<bf16_t, DH, 3>, grid, block, s, p);
    default: return hipErrorInvalidValue;  // more rows than the balanced path takes
  }
}

}  // namespace

hipError_t launch_attn_balanced(const AttnParams &p, int dh, hipStream_t s) {
  hipError_t e;
  if (dh == 64) e = launch_dh<64>(p, s);
  else if (dh == 96) e = launch_dh<96>(p, s);
  else e = launch_dh<128>(p, s);
  if (e != hipSuccess) return e;
  if (dh == 64) return launch_combine_dh<64>(p, s);
  if (dh == 96) return launch_combine_dh<96>(p, s);
  return launch_combine_dh<128>(p, s);
}

}  // namespace das
