// Launchers of the bfloat16 backward kernels, each in a translation unit of
// its own (the build script gives each source its flags): dK/dV on
// 16x16x32 MFMA in dkdv.hip (default machine scheduler), dQ in bwd.hip
// (iterative-ILP scheduler); the forward kernels, in attn.hip, keep the
// default scheduler.
#pragma once
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace attn {

// dK/dV tiles. 4-wave workgroups with several 16-key blocks per wave
// (every Q / dO operand read feeds one product per block): 32 keys per wave
// on 64-query steps at d = 32; 48 keys on 32-query steps at d = 64 and 32
// keys on 32-query steps at d = 128, where the fused form reads K from an
// LDS copy of the workgroup's 192 or 128 keys (30 or 36 KB) and the
// 32-query Q and dO stages leave room for two workgroups per CU. With 4
// waves, the two waves that share a SIMD come from two workgroups whose
// barriers are independent, so one can run its matrix products while the
// other waits or runs its softmax. The materialising form (no K; the staged
// block of the stored P instead) runs 32-key waves on 32-query tiles at
// d >= 64 (the fused tiling at d = 128; its P block reads need a
// power-of-two key block, so not the 48 keys of d = 64) and 16-key waves on
// 32-query tiles at d = 32. The atomic-dQ form uses 8 waves of 16 keys (its
// dQ tiling needs 8 waves).
constexpr int kDkv16BQ = 64;
constexpr int dkdv16_kb(int d, bool mat, bool aq) {
  return (aq || (mat && d < 64)) ? 1 : (d == 64 && !mat ? 3 : 2);
}
constexpr int dkdv16_nw(int d, bool mat, bool aq) { return aq ? 8 : 4; }
constexpr int dkdv16_bq(int d, bool mat) { return (mat || d >= 64) ? 32 : kDkv16BQ; }
constexpr int dkdv16_bkv(int d, bool mat, bool aq) { return 16 * dkdv16_kb(d, mat, aq) * dkdv16_nw(d, mat, aq); }
// queries per dQ workgroup (as in the forward)
constexpr int kDqBQ = 128;

// MAT: the backward of the materialising path; AQ: dQ by atomics (not
// instantiated in dkdv.hip: the atomic-dQ form is launched from attn.hip)
template <int D, bool CAUSAL, bool MAT, bool AQ>
void launch_dkdv16(BwdArgs a, int heads, hipStream_t st);

template <int D, bool CAUSAL, bool MAT>
void launch_dq16(BwdArgs a, int heads, hipStream_t st);

}  // namespace attn
