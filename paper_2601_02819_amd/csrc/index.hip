// Inverted selection index: for every (b, g, block t) the ascending list of
// query rows whose selection contains t (the transpose of sel), plus a table
// of attention work units (a unit = one block and up to unit_tokens entries of
// its list).  This lets the attention kernels run key-block-major: one K/V
// tile is loaded once and meets every query row that selected it.
//
// Entries are (row << 10) | (quarters << 6) | slot, where slot is the
// position of t among the row's entries (its sel vector, for 64-token blocks)
// and quarters is a 4-bit mask of the 16-key quarters of t the row attends
// to (all four for 64-token blocks).  The attention kernels store per-entry
// partial results in list order (contiguous per work unit); pmap[(row, slot)]
// = list position lets the per-row merges find them.
//
// Selections of m = 16 or 32 tokens, and rows whose local window goes to the
// band kernels, are indexed on 64-key tiles: the m-token blocks a row selected
// are grouped by the tile that holds them (tile = block / (64 / m)), and each
// tile entry carries the mask of the 16-key quarters its blocks cover.  The
// regrouping happens as the rows are read (row_entries), so the index is
// keyed by the tile geometry gm (m = 64, T = Lk / 64, ksel = min(Ksel, T) plus
// the band slot) while sel keeps its own width (the selection's Ksel).
//
// Integer-only passes, all deterministic (no order depends on timing):
//   count : per 256-row tile, an LDS bitmap [8 words][T] of who selected
//           what; popcounts give per-tile counts cntw[bg][w][t].
//   scan1 : per (bg, t), exclusive prefix over tiles -> cntw, total -> cnt,
//           and per 256 (bg, t) the sums of list lengths and units.
//   scan2 : one workgroup turns those sums into offsets; then per (bg, t)
//           the list offsets, unit offsets and the unit table.
//   fill  : rebuilds the tile bitmap; an entry's place in its list is
//           tile offset + number of lower rows in the tile that chose t.
#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool slot_valid(int t, int cur, int T) { return t >= 0 && t <= cur && t < T; }

// Width of a sel row: the selection's own Ksel (in its block units).
__device__ __forceinline__ int sel_width(const Geom &gm) { return gm.n_init + gm.window / gm.sm + 1 + gm.top_k; }

// Selections of 64-token blocks are indexed one thread per row: a row's
// entries are the valid prefix of its sel row (ascending causal blocks, ended
// by -1 or a block past the query's own), less its forced blocks when the
// band takes them.
__device__ __forceinline__ bool plain_rows(const Geom &gm) { return gm.sm == gm.m; }

// The forced blocks of Algorithm 1 for the query in block cur: the init blocks
// 0 .. ninit - 1 and the local window a_blk .. cur (a_blk >= ninit, so the
// two ranges are disjoint; both in selection blocks).  With the band, a row
// that holds all of them leaves them to the band kernels.
struct Forced {
  int ninit, a_blk, count;
  // wblk: the window in selection blocks (gm.window / gm.sm)
  __device__ __forceinline__ Forced(const Geom &gm, int cur, int wblk) {
    ninit = min(gm.n_init, cur + 1);
    a_blk = max(max(0, cur - wblk), ninit);
    count = ninit + cur - a_blk + 1;
  }
  __device__ __forceinline__ Forced(const Geom &gm, int cur) : Forced(gm, cur, gm.window / gm.sm) {}
  __device__ __forceinline__ bool has(int t) const { return t < ninit || t >= a_blk; }
};

// Selection block sizes of the attention entry points are 16, 32 or 64
// tokens, so the regrouping divides by shifts: sh = log2(sm), and a 64-key
// tile holds 64 >> sh blocks.  All fields are wave-uniform.
struct BlockShift {
  int sh, per_sh, qpb, wblk, nblk;
  __device__ __forceinline__ explicit BlockShift(const Geom &gm) {
    sh = __builtin_ctz((unsigned)gm.sm);
    per_sh = 6 - sh;
    qpb = gm.sm >> 4;
    wblk = gm.window >> sh;
    nblk = gm.Lk >> sh;
  }
};

// The regrouped entries of one row, one wave per row with lane s holding slot
// s of sel (t = that slot's block, -1 past the row's width).  A row's blocks
// are ascending, so a tile's blocks sit in adjacent lanes; a tile's first lane
// takes its slot by a ballot prefix count and ORs the quarters of the (at most
// 64 / m) lanes of its group.  With gm.band, a row holding every local block
// outside the init blocks (a_blk .. cur) leaves them to the band kernels
// (band_ok) together with its init blocks; other rows keep all their blocks.  A lane with `mine` set holds
// entry `pos` of the row: tile `tile` with quarter mask `qm`; n entries in all.
struct RowEntries {
  int tile;
  unsigned qm;
  int pos;
  int n;
  bool mine;
  bool band_ok;
};

// Whole-wave DPP shifts by one lane: lane i reads lane i - 1 (wave_shr:1) or
// lane i + 1 (wave_shl:1); a lane whose source is outside the wave reads 0.
__device__ __forceinline__ int from_lane_below(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x138, 0xF, 0xF, true);
}
__device__ __forceinline__ int from_lane_above(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x130, 0xF, 0xF, true);
}

// i: the row (wave-uniform).
__device__ __forceinline__ RowEntries row_entries(int t, int i, const Geom &gm, const BlockShift &bs) {
  const int lane = threadIdx.x & 63;
  RowEntries e;
  e.band_ok = false;
  const int cur = (gm.q_pos0 + i) >> bs.sh;
  const int per = 1 << bs.per_sh, qpb = bs.qpb;
  const bool in_range = t >= 0 && t <= cur && t < bs.nblk;
  const Forced f(gm, cur, bs.wblk);
  if (gm.band) e.band_ok = __popcll(__ballot(in_range && f.has(t))) == f.count;
  const bool valid = in_range && !(e.band_ok && f.has(t));
  const int tc = valid ? t >> bs.per_sh : -1;
  const unsigned qb = valid ? ((1u << qpb) - 1u) << ((t & (per - 1)) * qpb) : 0u;
  const int prev = from_lane_below(tc);
  const bool first = valid && (lane == 0 || prev != tc);
  const uint64_t heads = __ballot(first);
  e.pos = __popcll(heads & ((1ull << lane) - 1ull));
  e.n = __popcll(heads);
  unsigned acc = qb;
  int oq = (int)qb, otc = tc;  // the values of lane + dd
  for (int dd = 1; dd < per; ++dd) {
    oq = from_lane_above(oq);
    otc = from_lane_above(otc);
    if (lane + dd < 64 && otc == tc) acc |= (unsigned)oq;
  }
  e.mine = first && e.pos < gm.ksel - gm.band;
  e.tile = tc;
  e.qm = acc;
  return e;
}

// Sel rows a wave loads at once (regrouped rows), waited for together.  The
// fill stores as it goes, and loads and stores share one wait counter, so a
// load issued after a store cannot be waited for alone: each batch waits once
// for the previous batch's stores, not once per row.
constexpr int kRowBatch = 16;

// A plain row (one thread, its sel row staged at row[0 .. ks)) with the band:
// does it hold every forced block?
__device__ __forceinline__ bool plain_band_ok(const int32_t *row, int ks, int cur, const Geom &gm) {
  if (!gm.band) return false;
  const Forced f(gm, cur);
  int have = 0;
  for (int s = 0; s < ks; ++s) {
    const int t = row[s];
    if (!slot_valid(t, cur, gm.T)) break;
    have += f.has(t);
  }
  return have == f.count;
}

// The bitmap bm [8][T] of the 256-row tile w of (b, g) = bg: bit r % 32 of
// bm[r / 32][t] is set when row r has an entry for t.  Plain rows: the tile's
// sel rows, one contiguous run, are staged into rows_s ([kIndexTile][Ksel])
// with coalesced loads and each thread walks its row.  Regrouped rows: wave v
// takes rows 64v .. 64v + 63, one row per pass with its slots across the
// lanes (word-major bm, so a row's lanes, each on another t, hit different
// banks).  Every thread calls this (it holds barriers).
__device__ void build_tile_bitmap(uint32_t *bm, int32_t *rows_s, const int32_t *__restrict__ sel, const Geom &gm,
                                  int bg, int w) {
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ks = sel_width(gm);
  const int nrow = min(kIndexTile, gm.Lq - w * kIndexTile);
  const int64_t row0 = (int64_t)bg * gm.Lq + (int64_t)w * kIndexTile;
  for (int x = tid; x < gm.T * 8; x += 256) bm[x] = 0u;
  if (plain_rows(gm)) {
    const int32_t *src = sel + row0 * ks;
    for (int x = tid; x < nrow * ks; x += 256) rows_s[x] = src[x];
    __syncthreads();
    if (tid < nrow) {
      const int cur = (gm.q_pos0 + w * kIndexTile + tid) / gm.m;
      const bool bok = plain_band_ok(rows_s + tid * ks, ks, cur, gm);
      const Forced f(gm, cur);
      for (int s = 0; s < ks; ++s) {
        const int t = rows_s[tid * ks + s];
        if (!slot_valid(t, cur, gm.T)) break;
        if (!(bok && f.has(t))) atomicOr(&bm[(tid >> 5) * gm.T + t], 1u << (tid & 31));
      }
    }
    __syncthreads();
    return;
  }
  __syncthreads();
  const BlockShift bs(gm);
  for (int j0 = 0; j0 < 64; j0 += kRowBatch) {
    int t[kRowBatch];
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int r = wave * 64 + j0 + u;
      t[u] = (r < nrow && lane < ks) ? sel[(row0 + r) * ks + lane] : -1;
    }
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int r = wave * 64 + j0 + u;
      if (r < nrow) {  // wave-uniform
        const RowEntries e = row_entries(t[u], w * kIndexTile + r, gm, bs);
        if (e.mine) atomicOr(&bm[(r >> 5) * gm.T + e.tile], 1u << (r & 31));
      }
    }
  }
  __syncthreads();
}

// LDS of the count kernel (the fill kernel adds one list position per t).
// Plain rows stage their sel rows (width Ksel, in selection blocks) and, in
// the fill kernel, one band flag per row after them.
inline size_t index_lds_bytes(const Geom &g) {
  const bool plain = g.sm == g.m;
  const int ks = g.n_init + g.window / g.sm + 1 + g.top_k;
  return (size_t)g.T * 8 * sizeof(uint32_t) + (plain ? (size_t)kIndexTile * (ks + 1) * sizeof(int32_t) : 0);
}

__global__ __launch_bounds__(256) void index_count_kernel(const int32_t *__restrict__ sel, Geom gm, IndexWs ix) {
  extern __shared__ uint32_t bm[];
  const int w = blockIdx.x, bg = blockIdx.y;
  build_tile_bitmap(bm, reinterpret_cast<int32_t *>(bm + 8 * gm.T), sel, gm, bg, w);
  int32_t *dst = ix.cntw + ((int64_t)bg * ix.W + w) * gm.T;
  for (int t = threadIdx.x; t < gm.T; t += 256) {
    int c = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) c += __popc(bm[k * gm.T + t]);
    dst[t] = c;
  }
}

// The list scans.  For x = (b, g, t) with list length c: nu = ceil(c /
// unit_tokens) work units, and the flag f = (nu != 1) of the blocks whose
// dK/dV the finalize writes (from partial sums, or zeros for an empty list).
// Exclusive prefixes over x of c, nu and f give the list offsets, the unit
// offsets and the places in the finalize list.  Three passes, each x one
// thread: per 256 x the sums (with the tile scan), one workgroup's scan of
// those sums, then per 256 x the offsets and the unit table.
struct Counts3 {
  int c, nu, f;
};

__device__ __forceinline__ Counts3 list_counts(int c, int unit_tokens, bool live) {
  const int nu = (c + unit_tokens - 1) / unit_tokens;
  return Counts3{c, nu, live && nu != 1 ? 1 : 0};
}

// Exclusive scan of v over a 256-thread workgroup (c, nu and f each on its
// own); tot receives the workgroup's sums.  Holds barriers.
__device__ __forceinline__ Counts3 block_scan3(Counts3 v, Counts3 &tot) {
  __shared__ Counts3 wsum_s[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  Counts3 inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int a = __shfl_up(inc.c, d, 64), b = __shfl_up(inc.nu, d, 64), f = __shfl_up(inc.f, d, 64);
    if (lane >= d) {
      inc.c += a;
      inc.nu += b;
      inc.f += f;
    }
  }
  if (lane == 63) wsum_s[wave] = inc;
  __syncthreads();
  Counts3 pre{0, 0, 0};
  tot = Counts3{0, 0, 0};
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const Counts3 s = wsum_s[w];
    if (w < wave) {
      pre.c += s.c;
      pre.nu += s.nu;
      pre.f += s.f;
    }
    tot.c += s.c;
    tot.nu += s.nu;
    tot.f += s.f;
  }
  __syncthreads();  // wsum_s may be reused by the caller's next scan
  return Counts3{pre.c + inc.c - v.c, pre.nu + inc.nu - v.nu, pre.f + inc.f - v.f};
}

// Per (b, g, t): the tile counts become tile offsets (exclusive over the
// query tiles) and their total the list length; then the workgroup's sums.
__global__ __launch_bounds__(256) void index_scan_tiles_kernel(Geom gm, IndexWs ix, int nbgt) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  const bool live = x < nbgt;
  int run = 0;
  if (live) {
    const int bg = x / gm.T, t = x % gm.T;
    int32_t *col = ix.cntw + (int64_t)bg * ix.W * gm.T + t;
    // a batch of tiles' counts is loaded before any of them is overwritten (a
    // load behind a store waits for the store too: one round trip per batch)
    constexpr int U = 32;
    for (int w0 = 0; w0 < ix.W; w0 += U) {
      int c[U];
#pragma unroll
      for (int u = 0; u < U; ++u) c[u] = w0 + u < ix.W ? col[(int64_t)(w0 + u) * gm.T] : 0;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (w0 + u < ix.W) col[(int64_t)(w0 + u) * gm.T] = run;
        run += c[u];
      }
    }
    ix.cnt[x] = run;
  }
  Counts3 tot;
  block_scan3(list_counts(run, ix.unit_tokens, live), tot);
  if (threadIdx.x == 0) ix.wsum[blockIdx.x] = make_int4(tot.c, tot.nu, tot.f, 0);
}

// One workgroup: the workgroup sums become exclusive offsets (in place), and
// the totals (entries, units, finalize blocks) are written.
__global__ __launch_bounds__(256) void index_scan_sums_kernel(IndexWs ix, int nw, int nbgt) {
  Counts3 carry{0, 0, 0};
  for (int b0 = 0; b0 < nw; b0 += 256) {
    const int j = b0 + (int)threadIdx.x;
    const int4 v = j < nw ? ix.wsum[j] : make_int4(0, 0, 0, 0);
    Counts3 tot;
    const Counts3 ex = block_scan3(Counts3{v.x, v.y, v.z}, tot);
    if (j < nw) ix.wsum[j] = make_int4(carry.c + ex.c, carry.nu + ex.nu, carry.f + ex.f, 0);
    carry.c += tot.c;
    carry.nu += tot.nu;
    carry.f += tot.f;
  }
  if (threadIdx.x == 0) {
    ix.off[nbgt] = carry.c;
    ix.uoff[nbgt] = carry.nu;
    ix.totals[0] = carry.c;
    ix.totals[1] = carry.nu;
    ix.totals[2] = carry.f;
  }
}

// Per x: list offset, first unit, the unit table entries (block, first list
// entry) and, for nu != 1, the place in the finalize list (ascending x).
__global__ __launch_bounds__(256) void index_write_lists_kernel(IndexWs ix, int nbgt) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  const bool live = x < nbgt;
  const int c = live ? ix.cnt[x] : 0;
  const int4 base = ix.wsum[blockIdx.x];
  Counts3 tot;
  const Counts3 v = list_counts(c, ix.unit_tokens, live);
  const Counts3 ex = block_scan3(v, tot);
  if (!live) return;
  const int rb = base.y + ex.nu;
  ix.off[x] = base.x + ex.c;
  ix.uoff[x] = rb;
  for (int u = 0; u < v.nu; ++u) ix.units[rb + u] = make_int2(x, u * ix.unit_tokens);
  if (v.f) ix.fin[base.z + ex.f] = x;
}

// Writes each row's entries into their lists, its position-map row (list
// position per slot, -1 for empty slots, the band partial in the slot after the entries of
// a band row) and, with the band, its band flag.  The tile's first list
// position for each t (list offset + tile offset) is staged in LDS beside the
// bitmap; an entry's position adds the lower rows of the tile that chose t:
// the set bits of its own bitmap word below it plus those of the lower words,
// whose counts are staged per t as eight bytes (byte k: words 0 .. k - 1).
__global__ __launch_bounds__(256) void index_fill_kernel(const int32_t *__restrict__ sel, Geom gm, IndexWs ix) {
  extern __shared__ uint32_t bm[];
  uint64_t *pre_s = reinterpret_cast<uint64_t *>(bm + 8 * gm.T);
  int32_t *base_s = reinterpret_cast<int32_t *>(pre_s + gm.T);
  int32_t *rows_s = base_s + gm.T;  // plain rows: staged sel rows, then their list positions
  // Query tiles w, w + 1 of one (b, g) write adjacent runs of the same lists.
  // Workgroups are dealt to the 8 XCDs in turn (each XCD its own L2), so the
  // grid is renumbered to give each XCD one contiguous range of (bg, w): a
  // list's cache lines are then written through one L2.
  const int logical = xcd_item(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  const int w = logical % gridDim.x, bg = logical / gridDim.x, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int32_t *tile_off = ix.cntw + ((int64_t)bg * ix.W + w) * gm.T;
  const int32_t *list_off = ix.off + (int64_t)bg * gm.T;
  for (int t = tid; t < gm.T; t += 256) base_s[t] = list_off[t] + tile_off[t];
  build_tile_bitmap(bm, rows_s, sel, gm, bg, w);  // its barriers also publish base_s
  for (int t = tid; t < gm.T; t += 256) {
    uint64_t pre = 0;
    int run = 0;  // at most 7 x 32 = 224 rows below the last word
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      pre |= (uint64_t)run << (8 * k);
      run += __popc(bm[k * gm.T + t]);
    }
    pre_s[t] = pre;
  }
  __syncthreads();
  // rows of the tile below row r (word r / 32, bit r % 32) that chose t
  auto rank_of = [&](int t, int r) {
    const int word = r >> 5;
    return (int)((pre_s[t] >> (8 * word)) & 0xffu) + __popc(bm[word * gm.T + t] & ((1u << (r & 31)) - 1u));
  };
  const int ks = sel_width(gm);
  const int nrow = min(kIndexTile, gm.Lq - w * kIndexTile);
  const int64_t row0 = (int64_t)bg * gm.Lq + (int64_t)w * kIndexTile;
  if (plain_rows(gm)) {
    // entries take slots 0 .. n - 1 of the row's position-map row and the band
    // partial of a band row slot n, so that the merges' slot bound stays at the
    // row's own partial count; flag_s holds that slot (-1: no band partial)
    int32_t *flag_s = rows_s + kIndexTile * ks;
    const int i = w * kIndexTile + tid;
    if (tid < nrow) {
      const int cur = (gm.q_pos0 + i) / gm.m;
      const bool bok = plain_band_ok(rows_s + tid * ks, ks, cur, gm);
      const Forced f(gm, cur);
      int n = 0;
      for (int s = 0; s < ks; ++s) {  // the valid prefix, less the band's blocks
        const int t = rows_s[tid * ks + s];
        if (!slot_valid(t, cur, gm.T)) break;
        if (bok && f.has(t)) continue;
        const int32_t p = base_s[t] + rank_of(t, tid);
        ix.tok[p] = (i << 10) | (15 << 6) | n;
        rows_s[tid * ks + n] = p;  // n <= s: the slots still to be read are above
        ++n;
      }
      for (int s = n; s < ks; ++s) rows_s[tid * ks + s] = -1;
      flag_s[tid] = bok ? n : -1;
    }
    __syncthreads();
    // the tile's rows are consecutive, so their position-map rows form one contiguous run
    const int ksel = gm.ksel, nsp = ksel - gm.band;  // nsp <= ks slots for entries
    int32_t *dst = ix.pmap + row0 * ksel;
    for (int x = tid; x < nrow * ksel; x += 256) {
      const int r = x / ksel, s = x - r * ksel;
      dst[x] = s == flag_s[r] ? (int32_t)(ix.band_base + row0 + r) : s < nsp ? rows_s[r * ks + s] : -1;
    }
    if (gm.band && tid < nrow) ix.bflag[row0 + tid] = (uint8_t)(flag_s[tid] >= 0);
    return;
  }
  unsigned flag = 0;  // band flag of row 64 * wave + lane
  const BlockShift bs(gm);
  for (int j0 = 0; j0 < 64; j0 += kRowBatch) {
    int t[kRowBatch];
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int r = wave * 64 + j0 + u;
      t[u] = (r < nrow && lane < ks) ? sel[(row0 + r) * ks + lane] : -1;
    }
    // one wait for the whole batch here, before any branch: an (empty) use of
    // every loaded value, so that no row below waits on the stores again
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) asm volatile("" ::"v"(t[u]));
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int r = wave * 64 + j0 + u;
      if (r >= nrow) continue;  // wave-uniform
      const int i = w * kIndexTile + r;
      const int64_t x = row0 + r;
      const RowEntries e = row_entries(t[u], i, gm, bs);
      int32_t p = -1;
      if (e.mine) {
        p = base_s[e.tile] + rank_of(e.tile, r);
        ix.tok[p] = (i << 10) | ((int)(e.qm & 15u) << 6) | e.pos;
      }
      // entry pos's list position moves to lane pos (a lane below n has exactly
      // one sender; the others send to lane 63, which is below n only when all
      // 64 lanes are entries), so the row's position-map row is one store
      const int moved = __builtin_amdgcn_ds_permute((e.mine ? e.pos : 63) << 2, p);
      if (lane < gm.ksel)
        ix.pmap[x * gm.ksel + lane] =
            lane < e.n ? moved : (gm.band && e.band_ok && lane == e.n) ? (int32_t)(ix.band_base + x) : -1;
      if (lane == j0 + u) flag = e.band_ok ? 1u : 0u;
    }
  }
  if (gm.band && wave * 64 + lane < nrow) ix.bflag[row0 + wave * 64 + lane] = (uint8_t)flag;
}

hipError_t launch_build_index(const Geom &g, const int32_t *sel, const IndexWs &ix, hipStream_t s) {
  // Each launch's status is taken right after it: the attention kernels gather
  // through these lists, so a failed pass must stop the chain before them.
  hipError_t e;
  const int nbgt = g.B * g.Hkv * g.T;
  const size_t lds = index_lds_bytes(g);
  timing_begin("phsa_index_count", s);
  hipLaunchKernelGGL(index_count_kernel, dim3(ix.W, g.B * g.Hkv), dim3(256), lds, s, sel, g, ix);
  timing_end(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int nw = (nbgt + 255) / 256;  // list-scan workgroups (ix.wsum entries)
  timing_begin("phsa_index_scan_tiles", s);
  hipLaunchKernelGGL(index_scan_tiles_kernel, dim3(nw), dim3(256), 0, s, g, ix, nbgt);
  timing_end(s);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  timing_begin("phsa_index_scan_lists", s);
  hipLaunchKernelGGL(index_scan_sums_kernel, dim3(1), dim3(256), 0, s, ix, nw, nbgt);
  if ((e = hipGetLastError()) == hipSuccess)
    hipLaunchKernelGGL(index_write_lists_kernel, dim3(nw), dim3(256), 0, s, ix, nbgt);
  timing_end(s);
  if (e != hipSuccess || (e = hipGetLastError()) != hipSuccess) return e;
  timing_begin("phsa_index_fill", s);
  hipLaunchKernelGGL(index_fill_kernel, dim3(ix.W, g.B * g.Hkv), dim3(256),
                     lds + (size_t)g.T * (sizeof(int32_t) + sizeof(uint64_t)), s, sel,
                     g, ix);
  timing_end(s);
  return hipGetLastError();
}

}  // namespace phsa
