// Launches of the bfloat16 dK/dV kernel (dkdv16_kernel), fused and
// materialising forms. A translation unit of its own, compiled with the
// default machine scheduler: with the 32- and 48-key waves the dK/dV kernel
// runs about 2 % faster under it than under the iterative-ILP strategy that
// the dQ kernel keeps (bwd.hip). The atomic-dQ form is launched from
// attn.hip.
#include "launch.hpp"

namespace attn {

template <int D, bool CAUSAL, bool MAT, bool AQ>
void launch_dkdv16(BwdArgs a, int heads, hipStream_t st) {
  constexpr int kb = dkdv16_kb(D, MAT, AQ), nw = dkdv16_nw(D, MAT, AQ), bq = dkdv16_bq(D, MAT);
  constexpr int bkv = 16 * kb * nw;
  a.ntiles = (a.n + bkv - 1) / bkv;
  a.nblocks = heads * a.ntiles;
  hipLaunchKernelGGL((dkdv16_kernel<D, CAUSAL, nw, bq, MAT, AQ, kb>), dim3(a.nblocks), dim3(64 * nw), 0, st, a);
}

#define ATTN_DKDV16_INST(D, C)                                                \
  template void launch_dkdv16<D, C, false, false>(BwdArgs, int, hipStream_t); \
  template void launch_dkdv16<D, C, true, false>(BwdArgs, int, hipStream_t);

ATTN_DKDV16_INST(32, false)
ATTN_DKDV16_INST(32, true)
ATTN_DKDV16_INST(64, false)
ATTN_DKDV16_INST(64, true)
ATTN_DKDV16_INST(128, false)
ATTN_DKDV16_INST(128, true)

#undef ATTN_DKDV16_INST

}  // namespace attn
