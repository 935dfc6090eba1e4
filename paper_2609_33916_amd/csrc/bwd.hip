// Launches of the bfloat16 dQ kernel (fused and materialising forms).
// Compiled as a separate translation unit with the iterative-ILP machine
// scheduler (the build script gives each source its flags); the dK/dV
// launches live in dkdv.hip.
#include "launch.hpp"

namespace attn {

template <int D, bool CAUSAL, bool MAT>
void launch_dq16(BwdArgs a, int heads, hipStream_t st) {
  a.ntiles = (a.n + kDqBQ - 1) / kDqBQ;
  a.nblocks = heads * a.ntiles;
  hipLaunchKernelGGL((dq_kernel<bf16, D, CAUSAL, MAT>), dim3(a.nblocks), dim3(256), 0, st, a);
}

#define ATTN_BWD16_INST(D, C)                                                 \
  template void launch_dq16<D, C, false>(BwdArgs, int, hipStream_t);          \
  template void launch_dq16<D, C, true>(BwdArgs, int, hipStream_t);

ATTN_BWD16_INST(32, false)
ATTN_BWD16_INST(32, true)
ATTN_BWD16_INST(64, false)
ATTN_BWD16_INST(64, true)
ATTN_BWD16_INST(128, false)
ATTN_BWD16_INST(128, true)

#undef ATTN_BWD16_INST

}  // namespace attn
