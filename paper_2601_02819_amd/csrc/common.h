// Device helpers shared by the PHSA kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace phsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // storage type of bfloat16 values
// 16 raw bytes as a native vector: loads and stores of it are single values
// (a uint4 struct copy can be lowered to a memcpy through scratch memory)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}

// float -> bfloat16, round to nearest even (the gfx950 conversion instruction).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t x) { return bf16_to_f32(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f32_to_bf16(x); }

// 16x16x32 bf16 MFMA, fp32 accumulate.  Operand layout used throughout:
//   A (16 x 32, row-major M x K): lane l holds A[l % 16][8 * (l / 16) + 0..7]
//   B (32 x 16, K x N):           lane l holds B[8 * (l / 16) + 0..7][l % 16]
//   C (16 x 16):                  lane l holds C[4 * (l / 16) + 0..3][l % 16]
// A and B always use the same K assignment, so the contraction is exact
// whatever order the unit sums K in.
__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8 &a, const bf16x8 &b, const f32x4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 16-byte load of data that is read once (bypasses cache retention).
__device__ __forceinline__ uint4 ld_stream16(const bf16_t *p) {
  const uint32_t *q = reinterpret_cast<const uint32_t *>(p);
  return make_uint4(__builtin_nontemporal_load(q), __builtin_nontemporal_load(q + 1),
                    __builtin_nontemporal_load(q + 2), __builtin_nontemporal_load(q + 3));
}

// Stores of partial results that only a later merge kernel reads: non-temporal,
// so that they do not displace the gathered rows and key tiles that the
// writing kernel reuses (16-byte aligned).
__device__ __forceinline__ void st_stream16(bf16_t *dst, const bf16_t *src_lds) {
  __builtin_nontemporal_store(*reinterpret_cast<const u32x4 *>(src_lds), reinterpret_cast<u32x4 *>(dst));
}
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void st_stream_f2(float2 *dst, float a, float b) {  // one 8-byte store
  __builtin_nontemporal_store(f32x2{a, b}, reinterpret_cast<f32x2 *>(dst));
}

__device__ __forceinline__ bf16x8 load_bf16x8(const bf16_t *p) {  // 16-byte aligned
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(p));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Cross-row lane exchange with the gfx950 permlane swaps (VALU, no LDS
// round trip).  v_permlane16_swap exchanges the odd 16-lane rows of its first
// operand with the even rows of its second, v_permlane32_swap the upper half of
// the first with the lower half of the second; with x in both operands every
// lane ends up holding x of itself and of lane l ^ 16 (resp. l ^ 32), in an
// order that differs between the two lanes.  Commutative reductions of the
// pair are therefore equal in both lanes.
__device__ __forceinline__ float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;

// Column reads from a row-major bf16 LDS tile X (row pitch `pitch` elements)
// with the gfx950 transposing LDS load (ds_read_b64_tr_b16).  Within each
// 16-lane group the instruction hands lane j element (j % 4) of the 8 bytes
// addressed by lane 4e + j / 4, e = 0..3; giving lane i the address of
// X[r0 + i / 4][c0 + 4 (i % 4)] therefore delivers X[r0 + e][c0 + j] to lane j.
// r0 and c0 may differ between the four groups.  Rows must be 8-byte aligned.
__device__ __forceinline__ v4i16 lds_col4(const bf16_t *X, int pitch, int r0, int c0, int l16) {
  const bf16_t *p = X + (r0 + (l16 >> 2)) * pitch + c0 + 4 * (l16 & 3);
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)p);
}

// 8-element column fragment: lane j gets X[r0 + 0..3][c0 + j] then X[r1 + 0..3][c0 + j].
__device__ __forceinline__ bf16x8 lds_col8(const bf16_t *X, int pitch, int r0, int r1, int c0, int l16) {
  const v4i16 a = lds_col4(X, pitch, r0, c0, l16);
  const v4i16 b = lds_col4(X, pitch, r1, c0, l16);
  const v8i16 c = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, c);
}

// The partials of one (b, g, query row) for the per-row merges.  Half a wave
// owns a row: lane l32 reads the list positions of slots l32 and l32 + 32
// (-1 marks a slot without a partial).  slots() is a wave-uniform bound on the
// highest used slot of either half, and pos(s) gives each lane its own half's
// position of slot s (every lane must call it, s uniform).
struct RowSlots {
  int pa, pb;
  uint64_t valid;  // this half's slots that hold a partial
  uint32_t lo, hi; // slots < 32 / >= 32 used by either half
  __device__ __forceinline__ RowSlots(const int32_t *pmap, int64_t base, bool row_ok, int ksel, int half, int l32)
      : RowSlots((row_ok && l32 < ksel) ? pmap[base + l32] : -1, (row_ok && l32 + 32 < ksel) ? pmap[base + l32 + 32] : -1,
                 half) {}
  RowSlots() = default;
  // from the two positions this lane loaded (-1 for none), e.g. one row ahead
  __device__ __forceinline__ RowSlots(int pa_, int pb_, int half) : pa(pa_), pb(pb_) {
    const uint64_t ba = __ballot(pa >= 0), bb = __ballot(pb >= 0);
    valid = ((ba >> (32 * half)) & 0xffffffffull) | (((bb >> (32 * half)) & 0xffffffffull) << 32);
    lo = (uint32_t)ba | (uint32_t)(ba >> 32);
    hi = (uint32_t)bb | (uint32_t)(bb >> 32);
  }
  __device__ __forceinline__ int slots() const { return hi ? 64 - __clz(hi) : 32 - __clz(lo); }
  __device__ __forceinline__ int pos(int s, int half) const {
    const int src = half * 32 + (s & 31);
    return s < 32 ? __shfl(pa, src, 64) : __shfl(pb, src, 64);
  }
};

// Folds one partial of a row into a running merge (M, L, a) of Eq. 10-11:
// q = (m, l) in log2 units, raw = 8 bf16 features of its unnormalised O.  The
// maximum moves to the larger m and both sides are rescaled; a partial with
// m = -inf (no key) is skipped.
__device__ __forceinline__ void fold_partial(float &M, float &L, float (&a)[8], float2 q, const uint4 &raw) {
  if (q.x == -INFINITY) return;
  const float mn = fmaxf(M, q.x);
  const float sc = __builtin_amdgcn_exp2f(M - mn), w = __builtin_amdgcn_exp2f(q.x - mn);
  L = fmaf(w, q.y, L * sc);
  const bf16_t *pv = reinterpret_cast<const bf16_t *>(&raw);
#pragma unroll
  for (int j = 0; j < 8; ++j) a[j] = fmaf(w, bf16_to_f32(pv[j]), a[j] * sc);
  M = mn;
}

// The dispatcher hands workgroups to the 8 XCDs (each with its own L2) in
// turn by linear id.  Returns the work item of linear id `lin` (of n) such that
// each XCD takes one contiguous run of items: neighbouring items, which read
// the same tiles, then share an L2.  A bijection of 0..n-1.
__device__ __forceinline__ int xcd_item(int lin, int n) {
  const int x = lin & 7, j = lin >> 3;
  int off = 0;
  for (int y = 0; y < x; ++y) off += (n - y + 7) >> 3;  // items of the XCDs before
  return off + j;
}

// The exponentials of the softmax weights use the hardware 2^x instruction
// (__builtin_amdgcn_exp2f): its arguments are <= 0 or a bounded offset, and it
// flushes results below 2^-126, which are negligible against a sum >= 1.

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// fences global and private memory, and values held in registers across it
// (loads issued before the barrier, stored to LDS after it) can then be sent
// through scratch memory; this barrier leaves them in registers.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Orders a wave's LDS writes before its following LDS reads of other lanes'
// data.  A wave's LDS instructions execute in order, so this only has to stop
// the compiler from moving the accesses across it.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 64-row bf16 tiles in LDS without padding.  Row r holds D elements; its
// 16-byte chunk c sits at chunk position c ^ (r mod D / 8), which spreads the
// rows that one 16-lane group reads (row reads of MFMA operands and the
// transposing reads) over the LDS banks.  Element offset of (r, e):
template <int D>
__device__ __forceinline__ int swz(int r, int e) {
  return r * D + ((((e >> 3) ^ r) & (D / 8 - 1)) << 3) + (e & 7);
}

// 8-element column fragment of a swizzled tile (the layout of lds_col8).
template <int D>
__device__ __forceinline__ bf16x8 lds_col8_sw(const bf16_t *X, int r0, int r1, int c0, int l16) {
  const int e = c0 + 4 * (l16 & 3);
  const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(X + swz<D>(r0 + (l16 >> 2), e)));
  const v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(X + swz<D>(r1 + (l16 >> 2), e)));
  const v8i16 c = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, c);
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Copies a 64-row tile from global memory straight into LDS in the swizzled
// layout (global_load_lds: no registers, no LDS store instructions).  Each of
// the 4 waves issues D / 32 one-kilobyte copies; lane l of a copy lands at
// byte 16 l of it and fetches the chunk that belongs there.  Row r starts at
// element row_off(r) of src.  The copies count in vmcnt: each wave waits for
// vmcnt(0) and the workgroup then passes a barrier before the tile is read.
// wave must be wave-uniform (it selects the LDS destination).
template <int D, typename RowOff>
__device__ __forceinline__ void tile_dma(const bf16_t *src, RowOff row_off, bf16_t *dst, int wave, int lane) {
  constexpr int VPR = D / 8, RPI = 64 / VPR, NI = 64 / RPI / 4;
#pragma unroll
  for (int v = 0; v < NI; ++v) {
    const int blk = wave * NI + v, r = blk * RPI + lane / VPR, c = (lane % VPR) ^ (r & (VPR - 1));
    __builtin_amdgcn_global_load_lds(src + row_off(r) + c * 8, (lds_void_t *)(dst + blk * RPI * D), 16, 0, 0);
  }
}

// Waits until this wave's tile_dma copies have landed in LDS (vmcnt(0); the
// other counters are left alone).
__device__ __forceinline__ void dma_wait() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// Packs two 4-element float groups into a bf16 MFMA operand (elements 0..3,
// then 4..7), rounding to nearest even with the packed conversion instruction.
typedef float f32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ bf16x8 pack_bf16x8(const f32x4 &a, const f32x4 &b) {
  const f32x8 c = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_convertvector(c, bf16x8);
}

}  // namespace phsa
