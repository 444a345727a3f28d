// Device helpers shared by the direct-to-LDS GEMM kernels (gfx950):
// buffer resources, 16-byte global -> LDS copies, vmcnt waits, XOR-swizzled
// LDS regions and the MFMA 32x32x16 bf16 fragment reads from them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace pf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) void lds_void;

template <int I, int N, typename F>
__device__ __forceinline__ void sfor_impl(F &&f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    sfor_impl<I + 1, N>(f);
  }
}
template <int N, typename F>
__device__ __forceinline__ void sfor(F &&f) {
  sfor_impl<0, N>(f);
}

// Workgroups are dispatched round-robin over the 8 XCDs; remap so that
// consecutive logical ids run on the same XCD (and share its L2).
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  constexpr int X = 8;
  const int q = n / X, rem = n % X, x = bid % X, slot = bid / X;
  return x * q + min(x, rem) + slot;
}

// Buffer resource over [p, p + bytes): loads outside the range return zero
// (ragged token tiles, K padding).
__device__ __forceinline__ rsrc_t make_rsrc(const void *p, int64_t bytes) {
  const int64_t b = bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)b, 0x00020000);
}

// One 1 KiB window: lane i copies 16 bytes from rsrc + voff + soff to
// lds + 16 i.
// AUX: the copy's cache policy bits (0: default; 2: non-temporal, for an
// operand that one launch streams through once).
template <int AUX = 0>
__device__ __forceinline__ void dma16(rsrc_t r, uint8_t *lds, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)lds, 16, (int)voff, (int)soff, 0, AUX);
}

// Load of work-list metadata (tile lists, column and block indices) through
// the constant address space: these arrays do not change while a kernel
// runs, and such loads always use the scalar unit.  A generic load of them
// after an operand copy becomes a vector load (the copy counts as a
// possible writer), and its vmcnt wait then also waits for every copy in
// flight: the A copies of a step would land before its B copies issue.
template <typename T>
__device__ __forceinline__ T ld_meta(const T *p) {
  return *(const __attribute__((address_space(4))) T *)p;
}

// Wait until at most VM vector-memory operations of this wave are in flight
// and all of its LDS reads have returned.
template <int VM>
__device__ __forceinline__ void wait_vm() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4));
}
__device__ __forceinline__ void barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// XOR swizzle of the 16-byte chunk index in a [row][chunk] LDS region with
// CPR chunks per row (row-major operand, read with 16-byte fragment reads:
// 16 consecutive rows at a fixed chunk hit distinct banks).
template <int CPR>
__device__ __forceinline__ int swz_row(int r) {
  if constexpr (CPR == 4) return (r >> 2) & 3;
  else return (r >> 1) & 7;
}
// Same for a [k][n] region read with the transpose read (4 consecutive k
// rows x 32 bytes hit distinct banks).
template <int CPR>
__device__ __forceinline__ int swz_k(int k) {
  if constexpr (CPR == 4) return 0;
  else if constexpr (CPR == 8) return ((k >> 1) & 1) << 2;
  else return (k & 3) << 2;
}

// MFMA 32x32x16 operand (lane l: row l % 32, k = (l / 32) * 8 + 0..7 of
// k-slice kq) from a swizzled [row][chunk] region with row stride RB bytes.
template <int RB>
__device__ __forceinline__ bf16x8 frag_rows(const uint8_t *region, int r0, int kq, int lane) {
  constexpr int CPR = RB / 16;
  const int r = r0 + (lane & 31);
  const int c = kq * 2 + (lane >> 5);
  return *(const bf16x8 *)(region + r * RB + ((c ^ swz_row<CPR>(r)) << 4));
}

__device__ __forceinline__ s16x4 tr16(const uint8_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)(p));
}

// Same operand from a swizzled [k][n] region (n contiguous, RB bytes per k
// row): rows are n0 + l % 32, read with ds_read_b64_tr_b16 (within each
// 16-lane group, lanes 4m..4m+3 address k row m and lane j receives the 4
// k values of column j).  Each read's address is the region plus one
// integer offset: reads whose pointers are built up in several steps can
// reach the hardware without the alias information that tells them apart
// from copies still landing in another stage, and the compiler then waits
// for every copy in flight (the next step's included) before the read.
template <int RB>
__device__ __forceinline__ bf16x8 frag_kn(const uint8_t *region, int n0, int kq, int lane) {
  constexpr int CPR = RB / 16;
  const int g16 = lane >> 4, i = lane & 15;
  const int n = n0 + (g16 & 1) * 16 + (i & 3) * 4;
  const int k = kq * 16 + (g16 >> 1) * 8 + (i >> 2);
  const int c = n >> 3, half = ((n >> 2) & 1) << 3;
  const int off_lo = k * RB + ((c ^ swz_k<CPR>(k)) << 4) + half;
  const int off_hi = (k + 4) * RB + ((c ^ swz_k<CPR>(k + 4)) << 4) + half;
  const s16x4 lo = tr16(region + off_lo);
  const s16x4 hi = tr16(region + off_hi);
  const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Pipeline stage I of BYTES bytes: a distinct LDS object per stage, so that
// the compiler's LDS-DMA dependency tracking can tell the stages apart; only
// the stages a kernel uses are allocated.
template <int I, int BYTES>
__device__ __forceinline__ uint8_t *stage_buf() {
  __shared__ __attribute__((aligned(1024))) uint8_t buf[BYTES];
  return buf;
}

}  // namespace
}  // namespace pf
