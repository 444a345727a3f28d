// Pair blocks of b = 32 layouts.  With block rows and columns taken in
// aligned pairs, the kept 32 x 32 blocks group into 64 x 64 pair blocks, so
// the backward-data product and the weight gradient run on the 64-wide
// tiles of b = 64, whose steps read whole 128-byte row segments instead of
// half segments.  The gather builds each pair block (row-major [64][64]
// bf16) of W from the four blocks its source list names, zeros for dropped
// blocks; the scatter writes the kept quarters of pair-block gradients back
// to their blocks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pf_launch.h"

namespace pf {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// One workgroup per pair block: 64 rows x 8 chunks of 16 bytes, two chunks
// per thread.  src[4p + 2 a + h]: CSR position of the block in row half a,
// column half h (-1: zeros).
__global__ __launch_bounds__(256) void pair_gather_kernel(const uint16_t *__restrict__ W,
                                                          const int32_t *__restrict__ src,
                                                          uint16_t *__restrict__ Wp) {
  const int64_t p = blockIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int e = threadIdx.x + i * 256, row = e >> 3, ch = e & 7;
    const int32_t s = src[4 * p + (row >> 5) * 2 + (ch >> 2)];
    u32x4 v = {0u, 0u, 0u, 0u};
    if (s >= 0) v = *(const u32x4 *)(W + (int64_t)s * 1024 + (row & 31) * 32 + (ch & 3) * 8);
    *(u32x4 *)(Wp + p * 4096 + row * 64 + ch * 8) = v;
  }
}

// The inverse for the weight gradient computed on pair blocks: the kept
// blocks of each pair block (src >= 0) copied out to their CSR positions;
// dropped quarters are not written.
__global__ __launch_bounds__(256) void pair_scatter_kernel(const uint16_t *__restrict__ Wp,
                                                           const int32_t *__restrict__ src,
                                                           uint16_t *__restrict__ W) {
  const int64_t p = blockIdx.x;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int e = threadIdx.x + i * 256, row = e >> 3, ch = e & 7;
    const int32_t s = src[4 * p + (row >> 5) * 2 + (ch >> 2)];
    if (s >= 0)
      *(u32x4 *)(W + (int64_t)s * 1024 + (row & 31) * 32 + (ch & 3) * 8) =
          *(const u32x4 *)(Wp + p * 4096 + row * 64 + ch * 8);
  }
}

}  // namespace

hipError_t launch_pair_scatter(const void *Wp, const int32_t *src, int npair, void *W,
                               hipStream_t s) {
  if (npair <= 0) return hipSuccess;
  launch_kernel(pair_scatter_kernel, dim3((unsigned)npair), dim3(256), s, (const uint16_t *)Wp,
                src, (uint16_t *)W);
  return hipGetLastError();
}

hipError_t launch_pair_gather(const void *W, const int32_t *src, int npair, void *Wp,
                              hipStream_t s) {
  if (npair <= 0) return hipSuccess;
  launch_kernel(pair_gather_kernel, dim3((unsigned)npair), dim3(256), s, (const uint16_t *)W, src,
                (uint16_t *)Wp);
  return hipGetLastError();
}

}  // namespace pf
