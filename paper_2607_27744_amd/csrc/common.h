// Device-side helpers shared by the librocs kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rocs {

typedef __bf16 bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;   // MI355X: 8 accelerator complex dies, 32 CUs each

// D[16x16] += A[16x32] * B[32x16] on the matrix cores, bf16 in, fp32 out.
// Lane l holds A[l % 16][8 (l / 16) .. +7], B[8 (l / 16) .. +7][l % 16] and
// D[4 (l / 16) + i][l % 16] for i = 0..3.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// D[32x32] += A[32x16] * B[16x32], bf16 in, fp32 out (2x the work of the
// 16x16x32 shape per instruction and, on gfx950, about 2x its throughput).
// Lane l holds A[l % 32][8 (l / 32) .. +7], B[8 (l / 32) .. +7][l % 32] and
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] in element r = 0..15.
typedef float f32x16 __attribute__((ext_vector_type(16)));
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ u32x4 as_u32x4(bf16x8 v) { return __builtin_bit_cast(u32x4, v); }

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 r = {(bf16_t)a, (bf16_t)b};
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ float bf16_lo(uint32_t p) { return __builtin_bit_cast(float, p << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t p) { return __builtin_bit_cast(float, p & 0xffff0000u); }

template <typename T> __device__ __forceinline__ float load_f32(const T* p);
template <> __device__ __forceinline__ float load_f32<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_f32<bf16_t>(const bf16_t* p) { return (float)*p; }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return (bf16_t)x; }

// 16-byte global load that returns zeros when `ok` is false.
__device__ __forceinline__ u32x4 load16(const void* p, bool ok) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (ok) v = *reinterpret_cast<const u32x4*>(p);
  return v;
}

// Owner of candidate n under CSR offsets: the largest r in [0, R) with
// off[r] <= n. Empty requests (off[r] == off[r+1]) are skipped naturally.
__device__ __forceinline__ int owner_of(const int32_t* __restrict__ off, int R, int64_t n) {
  int lo = 0, hi = R - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if ((int64_t)off[mid] <= n) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Request tiling without a host-side pass over the offsets. Request r with
// c_r = off[r] candidate rows before it owns tile slots
//   g(r) = r + floor(c_r * rows_per_cand / TILE) ... g(r+1) - 1,
// at least max(1, ceil(n_r * rows_per_cand / TILE)) of them, and the slots of
// all requests are disjoint and below R + ceil(N * rows_per_cand / TILE). A
// workgroup given slot t finds its request by binary search and its tile
// index j = t - g(r); slots past the request's last tile exit at once.
__device__ __forceinline__ int64_t tile_base(const int32_t* __restrict__ off, int r,
                                             int rows_per_cand, int tile) {
  return (int64_t)r + ((int64_t)off[r] * rows_per_cand) / tile;
}

// The search is wave-parallel: each round the 64 lanes test 64 evenly spaced
// requests of the remaining range at once, and the ballot of the monotone
// test g(r) <= slot narrows the range 64-fold (two rounds of loads for up to
// 4096 requests instead of twelve dependent ones). Call it with every lane of
// the wave active; the result is wave-uniform.
__device__ __forceinline__ int request_of_slot(const int32_t* __restrict__ off, int R,
                                               int64_t slot, int rows_per_cand, int tile) {
  const int lane = (int)(threadIdx.x & 63);
  int lo = 0, n = R;                      // answer in [lo, lo + n); g(lo) <= slot holds
  while (n > 1) {
    const int step = (n + 63) / 64;
    const int r = lo + lane * step;
    const bool ok = r < lo + n && tile_base(off, r, rows_per_cand, tile) <= slot;
    const uint64_t m = __ballot(ok);      // lanes 0 .. k set, k the last request that fits
    const int k = 63 - __builtin_clzll(m);
    lo += k * step;
    n = min(step, n - k * step);
  }
  return __builtin_amdgcn_readfirstlane(lo);
}

// Workgroups are dispatched round-robin over the XCDs (workgroup b runs on
// XCD b % 8), and each XCD has its own L2. Renumber them so that consecutive
// logical indices run on the same XCD: work items that share operands
// (one candidate tile across output tiles, one request's K/V across candidate
// tiles) then hit the same L2. A bijection on [0, G).
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t G) {
  const uint32_t x = b % kNumXcd, i = b / kNumXcd;
  const uint32_t q = G / kNumXcd, rem = G % kNumXcd;
  return x * q + (x < rem ? x : rem) + i;
}

// Max / sum over lanes l and l ^ 32 (the two halves of the wave).
__device__ __forceinline__ float max_across_halves(float v) {
  const int iv = __builtin_bit_cast(int, v);
  auto s32 = __builtin_amdgcn_permlane32_swap(iv, iv, false, false);
  return fmaxf(__builtin_bit_cast(float, (int)s32[0]), __builtin_bit_cast(float, (int)s32[1]));
}

__device__ __forceinline__ float sum_across_halves(float v) {
  const int iv = __builtin_bit_cast(int, v);
  auto s32 = __builtin_amdgcn_permlane32_swap(iv, iv, false, false);
  return __builtin_bit_cast(float, (int)s32[0]) + __builtin_bit_cast(float, (int)s32[1]);
}

// Max over lanes l, l^16, l^32, l^48 (the four 16-lane rows of the wave).
__device__ __forceinline__ float max_across_rows(float v) {
  const int iv = __builtin_bit_cast(int, v);
  auto s16 = __builtin_amdgcn_permlane16_swap(iv, iv, false, false);
  v = fmaxf(__builtin_bit_cast(float, (int)s16[0]), __builtin_bit_cast(float, (int)s16[1]));
  const int jv = __builtin_bit_cast(int, v);
  auto s32 = __builtin_amdgcn_permlane32_swap(jv, jv, false, false);
  return fmaxf(__builtin_bit_cast(float, (int)s32[0]), __builtin_bit_cast(float, (int)s32[1]));
}

__device__ __forceinline__ float sum_across_rows(float v) {
  const int iv = __builtin_bit_cast(int, v);
  auto s16 = __builtin_amdgcn_permlane16_swap(iv, iv, false, false);
  v = __builtin_bit_cast(float, (int)s16[0]) + __builtin_bit_cast(float, (int)s16[1]);
  const int jv = __builtin_bit_cast(int, v);
  auto s32 = __builtin_amdgcn_permlane32_swap(jv, jv, false, false);
  return __builtin_bit_cast(float, (int)s32[0]) + __builtin_bit_cast(float, (int)s32[1]);
}

#define ROCS_LDS __attribute__((address_space(3)))
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Wait until at most N vector-memory operations of this wave are in flight
// (loads, stores and the LDS DMA loads all count there, and complete in
// issue order); LDS and export counters are not waited on.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until every LDS (and scalar-memory) operation of this wave is done.
__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));
}

// LDS byte address of a __shared__ object (wave-uniform).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const ROCS_LDS void*)p);
}

// 16 bytes per lane from global memory straight into LDS (the DMA form of
// global_load_dwordx4): lane i's bytes land at dst + 16 i, dst wave-uniform.
// Written as inline assembly on purpose: the compiler does not see an LDS
// write, so it adds no wait for these loads before unrelated LDS reads (its
// alias check would otherwise wait for every DMA load in flight before each
// LDS read of the ring). The caller orders LDS reads after the loads with
// wait_vmcnt and a barrier. The compiler does not count these loads either,
// which only makes its own vector-memory waits stricter. `dst` is an LDS
// byte address, wave-uniform.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t dst) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" :: "v"(src), "s"(dst) : "m0");
}
// Same with a wave-uniform base address and a 32-bit per-lane byte offset.
__device__ __forceinline__ void lds_dma16_sv(const void* sbase, uint32_t voff, uint32_t dst) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(sbase), "s"(dst) : "m0");
}

// LDS row swizzle for rows of D bf16 (2D bytes, D = 64 or 128) staged in
// their global layout: 16-byte chunk c of row `key` sits at chunk position
// c ^ kv_swizzle(key). Conflict-free for both read patterns: 16 consecutive
// rows at one chunk (row-major MFMA fragments) and 4 consecutive rows x 4
// consecutive chunks (transposing reads). Depends on key bits 0-3 only, so
// moving 16 rows keeps it, and chunk steps of 4 are an XOR of the offset.
template <int D>
__device__ __forceinline__ int kv_swizzle(int key) {
  static_assert(D == 64 || D == 128, "row width");
  if constexpr (D == 128) return ((key & 3) << 2) | ((key >> 2) & 3);
  else return (((key >> 1) & 1) << 2) | ((key >> 2) & 3);
}

// Workgroup barrier for the LDS ring. Each wave has waited for its own DMA
// loads before it arrives; the empty asm statements keep the compiler from
// moving LDS accesses across the barrier.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Buffer resource over `bytes` bytes from `base` (raw, untyped: the third
// word selects 32-bit data). A buffer load whose offset (VGPR offset plus
// immediate) reaches past `bytes` returns zero, and such a store is dropped,
// so a tile's edge needs no per-access branch.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

}  // namespace rocs
