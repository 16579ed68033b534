// Inverted selection index: for every (b, g, block t) the ascending list of
// query rows whose selection contains t (the transpose of sel), plus a table
// of attention work units (a unit = one block and up to unit_tokens entries of
// its list).  This lets the attention kernels run key-block-major: one K/V
// tile is loaded once and meets every query row that selected it.
//
// Entries are (row << 10) | (quarters << 6) | slot, where slot is the
// position of t in the row's sel vector and quarters is a 4-bit mask of the
// 16-key quarters of block t the row attends to (all four for 64-token
// blocks; see coarsen_kernel for smaller ones).  The attention kernels store
// per-entry partial results in list order (contiguous per work unit);
// pmap[(row, slot)] = list position lets the per-row merges find them.
//
// Four integer-only passes, all deterministic (no order depends on timing):
//   count : per 256-row tile, an LDS bitmap [T][256 bits] of who selected
//           what; popcounts give per-tile counts cntw[bg][w][t].
//   scan1 : per (bg, t), exclusive prefix over tiles -> cntw, total -> cnt.
//   scan2 : one workgroup scans cnt into list offsets and unit offsets and
//           writes the unit table.
//   fill  : rebuilds the tile bitmap; an entry's place in its list is
//           tile offset + number of lower rows in the tile that chose t.
#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool slot_valid(int t, int cur, int T) { return t >= 0 && t <= cur && t < T; }

// The tile's sel rows are one contiguous run: staged into rows_s
// ([kIndexTile][ksel]) with coalesced loads, then row tid is read from LDS.
__device__ void build_tile_bitmap(uint32_t *bm, int32_t *rows_s, const int32_t *sel, const Geom &gm, int bg, int w) {
  const int tid = threadIdx.x;
  for (int x = tid; x < gm.T * 8; x += 256) bm[x] = 0u;
  const int nrow = min(kIndexTile, gm.Lq - w * kIndexTile);
  const int32_t *src = sel + ((int64_t)bg * gm.Lq + (int64_t)w * kIndexTile) * gm.ksel;
  for (int x = tid; x < nrow * gm.ksel; x += 256) rows_s[x] = src[x];
  __syncthreads();
  if (tid < nrow) {
    const int cur = (gm.q_pos0 + w * kIndexTile + tid) / gm.m;
    // a row's valid slots are a prefix (ascending blocks, then -1 or blocks past cur)
    for (int s = 0; s < gm.ksel; ++s) {
      const int t = rows_s[tid * gm.ksel + s];
      if (!slot_valid(t, cur, gm.T)) break;
      atomicOr(&bm[t * 8 + (tid >> 5)], 1u << (tid & 31));
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(256) void index_count_kernel(const int32_t *__restrict__ sel, Geom gm, IndexWs ix) {
  extern __shared__ uint32_t bm[];
  const int w = blockIdx.x, bg = blockIdx.y;
  build_tile_bitmap(bm, reinterpret_cast<int32_t *>(bm + gm.T * 8), sel, gm, bg, w);
  int32_t *dst = ix.cntw + ((int64_t)bg * ix.W + w) * gm.T;
  for (int t = threadIdx.x; t < gm.T; t += 256) {
    int c = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) c += __popc(bm[t * 8 + k]);
    dst[t] = c;
  }
}

__global__ __launch_bounds__(256) void index_scan_tiles_kernel(Geom gm, IndexWs ix, int nbgt) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x >= nbgt) return;
  const int bg = x / gm.T, t = x % gm.T;
  int32_t *col = ix.cntw + (int64_t)bg * ix.W * gm.T + t;
  int run = 0;
  for (int w = 0; w < ix.W; ++w) {
    const int c = col[(int64_t)w * gm.T];
    col[(int64_t)w * gm.T] = run;
    run += c;
  }
  ix.cnt[x] = run;
}

// Single workgroup of 1024 threads: exclusive scans of list lengths and of
// units per list, then the unit table.
__global__ __launch_bounds__(1024) void index_scan_lists_kernel(Geom gm, IndexWs ix, int nbgt) {
  __shared__ int s_a[1024], s_b[1024];
  const int tid = threadIdx.x;
  const int per = (nbgt + 1023) / 1024;
  const int lo = min(nbgt, tid * per), hi = min(nbgt, lo + per);
  const int U = ix.unit_tokens;
  int sa = 0, sb = 0;
  for (int x = lo; x < hi; ++x) {
    const int c = ix.cnt[x];
    sa += c;
    sb += (c + U - 1) / U;
  }
  s_a[tid] = sa;
  s_b[tid] = sb;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {  // inclusive Hillis-Steele scan
    const int va = tid >= o ? s_a[tid - o] : 0;
    const int vb = tid >= o ? s_b[tid - o] : 0;
    __syncthreads();
    s_a[tid] += va;
    s_b[tid] += vb;
    __syncthreads();
  }
  int ra = s_a[tid] - sa, rb = s_b[tid] - sb;
  for (int x = lo; x < hi; ++x) {
    const int c = ix.cnt[x];
    const int nu = (c + U - 1) / U;
    ix.off[x] = ra;
    ix.uoff[x] = rb;
    for (int u = 0; u < nu; ++u) ix.units[rb + u] = make_int2(x, u * U);
    ra += c;
    rb += nu;
  }
  if (tid == 1023) {
    ix.off[nbgt] = s_a[1023];
    ix.uoff[nbgt] = s_b[1023];
    ix.totals[0] = s_a[1023];
    ix.totals[1] = s_b[1023];
  }
}

__global__ __launch_bounds__(256) void index_fill_kernel(const int32_t *__restrict__ sel,
                                                         const uint8_t *__restrict__ quarters, Geom gm, IndexWs ix) {
  extern __shared__ uint32_t bm[];
  // [kIndexTile][ksel]: the staged sel rows, each entry replaced in place by its list position
  int32_t *pm = reinterpret_cast<int32_t *>(bm + gm.T * 8);
  const int w = blockIdx.x, bg = blockIdx.y, tid = threadIdx.x;
  build_tile_bitmap(bm, pm, sel, gm, bg, w);
  const int i = w * kIndexTile + tid;
  if (i < gm.Lq) {
    const int cur = (gm.q_pos0 + i) / gm.m;
    const int32_t *tile_off = ix.cntw + ((int64_t)bg * ix.W + w) * gm.T;
    const int word = tid >> 5;
    const uint32_t below = (1u << (tid & 31)) - 1u;
    int s = 0;
    for (; s < gm.ksel; ++s) {  // the valid prefix
      const int t = pm[tid * gm.ksel + s];
      if (!slot_valid(t, cur, gm.T)) break;
      int rank = __popc(bm[t * 8 + word] & below);
      for (int k = 0; k < word; ++k) rank += __popc(bm[t * 8 + k]);
      const int32_t pos = ix.off[bg * gm.T + t] + tile_off[t] + rank;
      const int qm = quarters ? quarters[((int64_t)bg * gm.Lq + i) * gm.ksel + s] & 15 : 15;
      ix.tok[pos] = (i << 10) | (qm << 6) | s;
      pm[tid * gm.ksel + s] = pos;
    }
    // the last slot of a band geometry marks (-2) a row whose local window is in the band
    const bool in_band = ix.bflag && pm[tid * gm.ksel + gm.ksel - 1] == -2;
    for (; s < gm.ksel; ++s) pm[tid * gm.ksel + s] = -1;
    if (in_band) pm[tid * gm.ksel + gm.ksel - 1] = (int32_t)(ix.band_base + (int64_t)bg * gm.Lq + i);
  }
  __syncthreads();
  // the tile's rows are consecutive, so their position-map rows form one contiguous run
  const int nrow = min(kIndexTile, gm.Lq - w * kIndexTile);
  int32_t *dst = ix.pmap + ((int64_t)bg * gm.Lq + (int64_t)w * kIndexTile) * gm.ksel;
  for (int x = tid; x < nrow * gm.ksel; x += 256) dst[x] = pm[x];
}

// Blocks of m = 16 or 32 tokens run on the 64-key attention tiles: the
// m-token blocks a row selected are grouped by the 64-token tile that holds
// them (tile = block / (64 / m)), and each tile gets the mask of the 16-key
// quarters its selected blocks cover.  gc is the tile geometry (m = 64,
// T = Lk / 64, ksel = min(Ksel, T): no row holds more tiles than that).
// One wave per row, lane s holding slot s (Ksel <= 64): the rows are ascending,
// so a tile's blocks sit in adjacent lanes; a tile's first lane finds its
// output slot by a ballot prefix count and ORs the quarters of the (at most
// 64 / m) lanes of its group.  Reads and writes are contiguous per row.
// With gc.band, a row that holds every local block outside the init blocks
// (a_blk .. cur) leaves them to the band kernels: they are not regrouped, the
// row's last slot holds -2 and bflag = 1.  Other rows keep all their blocks.
__global__ __launch_bounds__(256) void coarsen_kernel(const int32_t *__restrict__ sel, Geom g, Geom gc,
                                                      int32_t *__restrict__ csel, uint8_t *__restrict__ cq,
                                                      uint8_t *__restrict__ bflag) {
  const int lane = threadIdx.x & 63;
  const int64_t x = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // row (b, g, i)
  if (x >= (int64_t)g.B * g.Hkv * g.Lq) return;                    // whole wave
  const int i = (int)(x % g.Lq);
  const int cur = (g.q_pos0 + i) / g.m;
  const int per = 64 / g.m, qpb = g.m / 16;
  const int t = lane < g.ksel ? sel[x * g.ksel + lane] : -1;
  const bool in_range = t >= 0 && t <= cur && t < g.T;
  bool band_ok = false;
  int a_blk = cur + 1;
  if (gc.band) {
    a_blk = max(max(0, cur - g.window / g.m), min(g.n_init, cur + 1));
    const int have = __popcll(__ballot(in_range && t >= a_blk));
    band_ok = a_blk <= cur && have == cur - a_blk + 1;
  }
  const bool valid = in_range && !(band_ok && t >= a_blk);
  const int tc = valid ? t / per : -1;
  const unsigned qb = valid ? ((1u << qpb) - 1u) << ((t % per) * qpb) : 0u;
  const int prev = __shfl_up(tc, 1, 64);
  const bool first = valid && (lane == 0 || prev != tc);
  const uint64_t heads = __ballot(first);
  const int pos = __popcll(heads & ((1ull << lane) - 1ull));
  const int n = __popcll(heads);
  unsigned acc = qb;
  for (int dd = 1; dd < per; ++dd) {
    const unsigned o = __shfl_down(qb, dd, 64);
    const int otc = __shfl_down(tc, dd, 64);
    if (lane + dd < 64 && otc == tc) acc |= o;
  }
  int32_t *out = csel + x * gc.ksel;
  uint8_t *oq = cq + x * gc.ksel;
  if (first && pos < gc.ksel - gc.band) {
    out[pos] = tc;
    oq[pos] = (uint8_t)acc;
  }
  if (lane >= n && lane < gc.ksel) {
    out[lane] = (gc.band && band_ok && lane == gc.ksel - 1) ? -2 : -1;
    oq[lane] = 0;
  }
  if (gc.band && lane == 0) bflag[x] = band_ok ? 1 : 0;
}

hipError_t launch_coarsen(const Geom &g, const Geom &gc, const int32_t *sel, int32_t *csel, uint8_t *cq,
                          uint8_t *bflag, hipStream_t s) {
  const int64_t nrows = (int64_t)g.B * g.Hkv * g.Lq;
  timing_begin("phsa_coarsen", s);
  hipLaunchKernelGGL(coarsen_kernel, dim3((unsigned)((nrows + 3) / 4)), dim3(256), 0, s, sel, g, gc, csel, cq, bflag);
  timing_end(s);
  return hipGetLastError();
}

hipError_t launch_build_index(const Geom &g, const int32_t *sel, const uint8_t *quarters, const IndexWs &ix,
                              hipStream_t s) {
  const int nbgt = g.B * g.Hkv * g.T;
  const size_t lds = (size_t)g.T * 8 * sizeof(uint32_t);
  const size_t rows_lds = (size_t)kIndexTile * g.ksel * sizeof(int32_t);
  timing_begin("phsa_index_count", s);
  hipLaunchKernelGGL(index_count_kernel, dim3(ix.W, g.B * g.Hkv), dim3(256), lds + rows_lds, s, sel, g, ix);
  timing_end(s);
  timing_begin("phsa_index_scan_tiles", s);
  hipLaunchKernelGGL(index_scan_tiles_kernel, dim3((nbgt + 255) / 256), dim3(256), 0, s, g, ix, nbgt);
  timing_end(s);
  timing_begin("phsa_index_scan_lists", s);
  hipLaunchKernelGGL(index_scan_lists_kernel, dim3(1), dim3(1024), 0, s, g, ix, nbgt);
  timing_end(s);
  timing_begin("phsa_index_fill", s);
  hipLaunchKernelGGL(index_fill_kernel, dim3(ix.W, g.B * g.Hkv), dim3(256), lds + rows_lds, s, sel, quarters, g, ix);
  timing_end(s);
  return hipGetLastError();
}

}  // namespace phsa
