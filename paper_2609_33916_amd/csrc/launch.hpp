// Launchers of the bfloat16 backward kernels (dK/dV on 16x16x32 MFMA, dQ),
// defined in bwd.hip: a translation unit of its own, compiled with the
// iterative-ILP machine scheduler (the build script gives each source its
// flags), while the forward kernels keep the default scheduler.
#pragma once
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace attn {

// dK/dV tiles. The fused path runs 4-wave workgroups of 32 keys per wave
// (every Q / dO operand read feeds two products): 64 queries per step for
// d <= 64; 32 at d = 128, where K is read from an LDS copy of the
// workgroup's 128 keys (36 KB) and the 32-query Q and dO stages leave room
// for two workgroups per CU. With 4 waves, the two waves that share a SIMD
// come from two workgroups whose barriers are independent, so one can run its
// matrix products while the other waits or runs its softmax. The
// materialising form at d = 128 and the atomic-dQ form use 8 waves of 16
// keys (their extra LDS tiles leave room for one workgroup per CU; the
// atomic form's dQ tiling needs 8 waves). For d <= 64 the materialising form
// runs 4-wave workgroups of 16-key waves on 32-query tiles (its LDS then
// leaves room for two workgroups per CU; at d = 128 the halved step measured
// slower).
constexpr int kDkv16BQ = 64;
constexpr int dkdv16_kb(int d, bool mat_or_aq) { return mat_or_aq ? 1 : 2; }
constexpr int dkdv16_nw(int d, bool mat, bool aq) { return (aq || (mat && d > 64)) ? 8 : 4; }
constexpr int dkdv16_bq(int d, bool mat) { return ((mat && d <= 64) || (!mat && d > 64)) ? 32 : kDkv16BQ; }
constexpr int dkdv16_bkv(int d, bool mat, bool aq) { return 16 * dkdv16_kb(d, mat || aq) * dkdv16_nw(d, mat, aq); }
// queries per dQ workgroup (as in the forward)
constexpr int kDqBQ = 128;

// MAT: the backward of the materialising path; AQ: dQ by atomics (not
// instantiated in bwd.hip: the atomic-dQ form is launched from attn.hip)
template <int D, bool CAUSAL, bool MAT, bool AQ>
void launch_dkdv16(BwdArgs a, int heads, hipStream_t st);

template <int D, bool CAUSAL, bool MAT>
void launch_dq16(BwdArgs a, int heads, hipStream_t st);

}  // namespace attn
