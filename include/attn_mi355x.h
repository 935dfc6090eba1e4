/*
 * attn_mi355x.h -- C ABI of the fused attention forward+backward library for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation is one attention layer over [B, H, n, d] tensors: the paper's
 * naive path materialises the n x n attention matrix A and reads it back,
 * the fused path consumes A as soon as it is produced (Fig. fig:concept,
 * section sec:dnf-onf-machines; Paper II, sections sec:paper2-cpu and
 * sec:paper2-gv-fix). This library is the fused path: no n x n buffer is ever
 * allocated or written, and each output element has a single writer (the
 * race-free restructuring of Paper II, section sec:paper2-crash, and the
 * per-key-column gradient pass of section sec:paper2-gv-fix), so no global
 * atomics are issued.
 *
 * Mathematics (per batch b and head h; s = scale):
 *   S = s Q K^T, masked to -inf where key j > query i when causal
 *   P = softmax_rows(S), L_i = ln sum_j exp(S_ij)       (natural log)
 *   O = P V
 *   dV = P^T dO, dP = dO V^T, D_i = sum_j P_ij dP_ij, dS = P * (dP - D)
 *   dQ = s dS K, dK = s dS^T Q
 * which is the gradient of <O, dO> with respect to Q, K, V.
 *
 * Layout. Q, K, V, dO, O, dQ, dK, dV are dense row-major [B, H, n, d]
 * (d fastest, no padding) in the element type `dtype`; L is float32 [B, H, n].
 * All device pointers; every tensor must be 16-byte aligned, L and the
 * workspace 4-byte aligned. Outputs must not alias inputs or each other.
 *
 * Ownership. The caller allocates and owns every buffer, including the
 * workspace. The library never allocates or frees memory, keeps no state
 * between calls and is safe to call from several host threads.
 *
 * Execution. Calls enqueue kernels on `stream` (a hipStream_t; NULL means
 * the default stream) and return without synchronising. Results are valid
 * once the stream reaches that point.
 *
 * Errors. Every entry point validates all arguments before touching the GPU;
 * on an invalid argument it returns the negative code below and launches
 * nothing. A launch failure reported by the HIP runtime returns ATTN_E_HIP.
 * Faults inside a running kernel surface as errors of later HIP calls.
 */
#ifndef ATTN_MI355X_H
#define ATTN_MI355X_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of Q, K, V, dO and of the outputs O, dQ, dK, dV. Arithmetic
 * accumulates in float32 in both cases. */
typedef enum {
  ATTN_BF16 = 0, /* bfloat16 inputs and outputs (round to nearest even) */
  ATTN_F32 = 1   /* float32 inputs and outputs */
} attn_dtype;

enum {
  ATTN_OK = 0,
  ATTN_E_NULL = -1,        /* a required pointer is NULL */
  ATTN_E_SHAPE = -2,       /* B, H or n < 1, or the problem is too large to index */
  ATTN_E_UNSUPPORTED = -3, /* d not in {32, 64, 128}, or unknown dtype */
  ATTN_E_ALIGN = -4,       /* a tensor is not 16-byte aligned (L/workspace: 4-byte) */
  ATTN_E_WORKSPACE = -5,   /* workspace_bytes < attn_workspace_bytes(B, H, n, d) */
  ATTN_E_HIP = -6,         /* the HIP runtime rejected a kernel launch */
  ATTN_E_ARG = -7          /* scale not finite, or causal not 0/1 */
};

/* Bytes of device workspace attn_fwd_bwd needs: two float32 per query row,
 * the backward's row pre-pass D_i = sum_j P_ij dP_ij (computed as
 * sum_c dO_ic O_ic) and the row log-sum-exp in base 2 (L_i log2 e), i.e.
 * 2*B*H*n*4 bytes. Returns 0 for non-positive sizes. */
size_t attn_workspace_bytes(int B, int H, int n, int d);

/* Forward only: O and L from Q, K, V (Paper I, section sec:paper1, with A
 * never stored). O is [B,H,n,d] in dtype, L float32 [B,H,n]. */
int attn_fwd(const void* Q, const void* K, const void* V, void* O, float* L,
             int B, int H, int n, int d, float scale, int causal, int dtype,
             void* stream);

/* Fused forward+backward (Paper II, the fused "Algorithm 2"): O, L, dQ, dK,
 * dV from Q, K, V, dO. `workspace` must hold attn_workspace_bytes(B,H,n,d)
 * bytes; its contents on entry are ignored and on exit are unspecified. */
int attn_fwd_bwd(const void* Q, const void* K, const void* V, const void* dO,
                 void* O, float* L, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int n, int d, float scale, int causal, int dtype,
                 void* stream);

/* Backward only (Paper II's "Algorithm 1" reads the forward's results back
 * from memory; here only the O(n) row statistics are): dQ, dK, dV from Q, K,
 * V, the forward's O and L, and dO. A pre-pass computes D_i = sum_c dO_ic O_ic
 * from the given O (in its stored precision) and the base-2 L into the
 * workspace (attn_workspace_bytes(B,H,n,d) bytes); then the dK/dV and dQ
 * kernels of attn_fwd_bwd run unchanged. O and L must be the forward's outputs
 * for the same Q, K, V, scale and mask. */
int attn_bwd(const void* Q, const void* K, const void* V, const void* O, const float* L,
             const void* dO, void* dQ, void* dK, void* dV,
             void* workspace, size_t workspace_bytes,
             int B, int H, int n, int d, float scale, int causal, int dtype,
             void* stream);

/* attn_fwd_bwd with per-kernel timing: when `events` is not NULL it must
 * point to 4 hipEvent_t created by the caller; events[0] is recorded on
 * `stream` before the forward kernel, events[1] after it, events[2] after the
 * dK/dV kernel and events[3] after the dQ kernel, so hipEventElapsedTime of
 * consecutive pairs gives each kernel's device time. Same arguments, results
 * and errors as attn_fwd_bwd otherwise (a failed event record returns
 * ATTN_E_HIP). */
int attn_fwd_bwd_timed(const void* Q, const void* K, const void* V, const void* dO,
                       void* O, float* L, void* dQ, void* dK, void* dV,
                       void* workspace, size_t workspace_bytes,
                       int B, int H, int n, int d, float scale, int causal, int dtype,
                       void* stream, void* const* events);

/* Static, NUL-terminated description of a status code (never NULL). */
const char* attn_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_MI355X_H */
