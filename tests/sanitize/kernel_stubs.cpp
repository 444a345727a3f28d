// Stand-ins for the kernel launchers in a host-only build of the C ABI
// (layout builder, argument checks, launch planning) under the address and
// undefined-behaviour sanitizers.  The driver never reaches a launch: every
// compute call it makes fails validation or finds its layout not uploaded.
// Reaching one aborts.
#include <cstdio>
#include <cstdlib>

#include "pf_internal.h"

namespace pf {

[[noreturn]] static void no_kernels(const char *f) {
  std::fprintf(stderr, "kernel launcher %s reached in the host-only build\n", f);
  std::abort();
}

hipError_t launch_nt(int, int, int, bool, int, const NTArgs &, hipStream_t) { no_kernels("nt"); }
template <int BLK, bool BKN>
hipError_t launch_ntd_bb(int, int, const NTArgs &, hipStream_t) {
  no_kernels("ntd");
}
template hipError_t launch_ntd_bb<32, false>(int, int, const NTArgs &, hipStream_t);
template hipError_t launch_ntd_bb<32, true>(int, int, const NTArgs &, hipStream_t);
template hipError_t launch_ntd_bb<64, false>(int, int, const NTArgs &, hipStream_t);
template hipError_t launch_ntd_bb<64, true>(int, int, const NTArgs &, hipStream_t);
template hipError_t launch_ntd_bb<128, false>(int, int, const NTArgs &, hipStream_t);
template hipError_t launch_ntd_bb<128, true>(int, int, const NTArgs &, hipStream_t);
hipError_t launch_reduce_rows(int, int, const float *, int64_t, int64_t, void *, int64_t,
                              hipStream_t) {
  no_kernels("reduce_rows");
}
hipError_t launch_tn(int, int, const TNArgs &, hipStream_t) { no_kernels("tn"); }
hipError_t launch_tnw(int, int, const TNArgs &, hipStream_t) { no_kernels("tnw"); }
hipError_t launch_tnw_reduce(int, int, const TNArgs &, hipStream_t) { no_kernels("tnw_reduce"); }
hipError_t launch_pair_gather(const void *, const int32_t *, int, void *, hipStream_t) {
  no_kernels("pair_gather");
}
hipError_t launch_pair_scatter(const void *, const int32_t *, int, void *, hipStream_t) {
  no_kernels("pair_scatter");
}
hipError_t launch_tn_reduce(int, int, const TNArgs &, hipStream_t) { no_kernels("tn_reduce"); }
hipError_t launch_skinny(bool, const SkinnyArgs &, hipStream_t) { no_kernels("skinny"); }
hipError_t launch_mix_dgamma(int, const void *, const void *, int64_t, const float *, int,
                             float *, float *, hipStream_t) {
  no_kernels("mix_dgamma");
}
hipError_t launch_gelu_bwd(int, int64_t, const void *, const void *, void *, hipStream_t) {
  no_kernels("gelu_bwd");
}
hipError_t launch_attn_fwd(const AttnArgs &, int, hipStream_t) { no_kernels("attn_fwd"); }
hipError_t launch_attn_bwd_dq(const AttnArgs &, int, hipStream_t) { no_kernels("attn_dq"); }
hipError_t launch_attn_bwd_dkv(const AttnArgs &, int, hipStream_t) { no_kernels("attn_dkv"); }
hipError_t attn_scratch(float **) { no_kernels("attn_scratch"); }
hipError_t launch_bfly(bool, const BflyArgs &, hipStream_t) { no_kernels("bfly"); }

}  // namespace pf
