// Launches of the bfloat16 backward kernels: dK/dV (dkdv16_kernel) and dQ.
// Compiled as a separate translation unit with its own scheduler flags; the
// instantiations below cover every (d, causal, variant) the C ABI dispatches
// except the atomic-dQ dK/dV kernel, which attn.hip launches itself.
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

template <int D, bool CAUSAL, bool MAT>
void launch_dq16(BwdArgs a, int heads, hipStream_t st) {
  a.ntiles = (a.n + kDqBQ - 1) / kDqBQ;
  a.nblocks = heads * a.ntiles;
  hipLaunchKernelGGL((dq_kernel<bf16, D, CAUSAL, MAT>), dim3(a.nblocks), dim3(256), 0, st, a);
}

#define ATTN_BWD16_INST(D, C)                                                 \
  template void launch_dkdv16<D, C, false, false>(BwdArgs, int, hipStream_t); \
  template void launch_dkdv16<D, C, true, false>(BwdArgs, int, hipStream_t);  \
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
