/*
 * attn_mi355x.h -- C ABI of the fused attention forward+backward library for
 * AMD Instinct MI355X (gfx950).
 *
 * The operation is one attention layer over [B, H, n, d] tensors: the paper's
 * naive path materialises the n x n attention matrix A and reads it back,
 * the fused path consumes A as soon as it is produced (Fig. fig:concept,
 * section sec:dnf-onf-machines; Paper II, sections sec:paper2-cpu and
 * sec:paper2-gv-fix). The attn_fwd / attn_fwd_bwd / attn_bwd entry points are
 * the fused path: no n x n buffer is ever allocated or written, and each
 * output element has a single writer (the race-free restructuring of Paper
 * II, section sec:paper2-crash, and the per-key-column gradient pass of
 * section sec:paper2-gv-fix), so no global atomics are issued. The attn_mat_*
 * entry points are the naive path on the same kernels' tiling, kept for the
 * paper's fused-versus-naive comparison: the forward writes A, the backward
 * reads it instead of recomputing it.
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
 *
 * Where this interface departs from the plain statement of the problem
 * (forward, backward and fused forward+backward over B x N x D arrays, Paper
 * II, section sec:paper2-cpu), on purpose:
 *  - `dtype` is passed as int (an attn_dtype value) and `stream` as void*
 *    (a hipStream_t): the same ABI, but the header needs no HIP include and
 *    foreign-function callers pass plain integers and pointers;
 *  - the workspace holds two float32 rows per query, not one: the D row and
 *    the base-2 log-sum-exp row, so the backward kernels read L already in
 *    the base their exponentials use (attn_workspace_bytes below);
 *  - ATTN_E_ARG reports a non-finite scale or a causal flag other than 0/1,
 *    which the other codes do not describe.
 * The paper defines none of attn_workspace_bytes, attn_strerror or the
 * status codes: they are part of this interface only.
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
  ATTN_E_WORKSPACE = -5,   /* workspace_bytes < attn_workspace_bytes(B, H, n, d), or
                              p_bytes < attn_mat_bytes(B, H, n, dtype) */
  ATTN_E_HIP = -6,         /* the HIP runtime rejected a kernel launch */
  ATTN_E_ARG = -7,         /* scale not finite, or causal not 0/1 */
  ATTN_E_SCRATCH = -8      /* attn_fwd_bwd_noalloc: B*H*n > attn_noalloc_max_rows() */
};

/* Not an operation of the paper: the size of the caller-owned scratch rows.
 * Bytes of device workspace attn_fwd_bwd needs: two float32 per query row,
 * the backward's row pre-pass D_i = sum_j P_ij dP_ij (computed as
 * sum_c dO_ic O_ic and stored negated, the value the backward's dP
 * accumulators start from) and the row log-sum-exp in base 2 (L_i log2 e),
 * i.e. 2*B*H*n*4 bytes. Returns 0 for non-positive sizes. */
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

/* ---- Without device allocation -----------------------------------------
 * For callers that cannot allocate device memory at call time: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc. attn_fwd_bwd_noalloc computes exactly what attn_fwd_bwd computes,
 * with the same kernels and bit-identical results, but takes no workspace:
 * the D and base-2 log-sum-exp rows live in a fixed 16 MiB device array of
 * the library (one per GPU, held from the first call on that GPU until the
 * process ends), so B*H*n may be at most attn_noalloc_max_rows() = 2097152
 * query rows (ATTN_E_SCRATCH otherwise; n = 16384 at 64 heads uses half of
 * it). The call allocates nothing and needs no zeroing: every scratch row is
 * written by the forward kernel before the backward kernels read it.
 * All calls on one GPU share that GPU's array and it keeps the last call's
 * contents: two calls that may run at the same time on one GPU (different
 * streams, or different host threads without ordering) race on it and give
 * wrong results; order them on one stream. The first call on a GPU looks the
 * array's address up (hipGetSymbolAddress) with that GPU current; a failed
 * lookup returns ATTN_E_HIP. Other arguments and errors as attn_fwd_bwd. */
size_t attn_noalloc_max_rows(void);

int attn_fwd_bwd_noalloc(const void* Q, const void* K, const void* V, const void* dO,
                         void* O, float* L, void* dQ, void* dK, void* dV,
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

/* ---- Atomic-dQ variant -------------------------------------------------
 * The alternative Paper II weighs against recomputation (sections
 * sec:paper2-atomics, sec:paper2-gk-fix): instead of a separate dQ kernel
 * that recomputes S and dP per query block, the dK/dV kernel also forms
 * dQ = dS K for its 128-key block and adds it to a float32 accumulator in
 * the workspace with atomic adds, B*H*n*d*ceil(n/128) of them without a mask
 * (about half that under the causal mask); a last pass writes
 * dQ = scale * accumulator in bfloat16. Same results as attn_fwd_bwd within
 * rounding; dQ's summation order depends on scheduling, so repeated calls
 * may differ in the last bits of dQ. bfloat16 only (ATTN_E_UNSUPPORTED for
 * float32). */

/* Workspace for attn_fwd_bwd_atomic: the float32 accumulator B*H*n*d*4
 * bytes, then the D and base-2 L rows (attn_workspace_bytes). The workspace
 * must be 16-byte aligned. 0 for invalid sizes. */
size_t attn_workspace_bytes_atomic(int B, int H, int n, int d);

/* Forward + backward with atomic dQ: zero the accumulator, forward, one
 * dK/dV/dQ kernel, finalize. Arguments as attn_fwd_bwd. */
int attn_fwd_bwd_atomic(const void* Q, const void* K, const void* V, const void* dO,
                        void* O, float* L, void* dQ, void* dK, void* dV,
                        void* workspace, size_t workspace_bytes,
                        int B, int H, int n, int d, float scale, int causal, int dtype,
                        void* stream);

/* ---- Naive (materialising) path --------------------------------------
 * The realisation the paper compares the fused one against: the forward
 * stores the attention matrix A = P (Table tab:paper1-dram counts it as the
 * n x n array written next to Out) and the backward reads P back instead of
 * recomputing it (Paper II, section sec:paper2-cpu, "Algorithm 1").
 *
 * P layout: [B, H, n, lda] in `dtype`, lda = n rounded up to a multiple of
 * 128; element (b, h, i, j) = P_ij for query i < n and key j < n. The forward
 * writes, per 32-query block, every 64-key tile that holds a key the block
 * sees (all tiles without a mask; under the causal mask the tiles up to the
 * diagonal), with zeros where masked; entries it does not write are left
 * untouched and never used. The caller allocates P (attn_mat_bytes
 * bytes, 16-byte aligned) and owns it.
 * Sizes: n <= 1048576 (ATTN_E_SHAPE otherwise). */

/* Bytes of the P buffer: B*H*n*lda*sizeof(dtype); 0 for invalid sizes. */
size_t attn_mat_bytes(int B, int H, int n, int dtype);

/* Naive forward: O, L and P from Q, K, V. Two sweeps over the key tiles per
 * query block: the first computes each row's log-sum-exp, the second writes
 * the normalised P and accumulates O = P V (for bf16, from P as stored). */
int attn_mat_fwd(const void* Q, const void* K, const void* V, void* O, float* L,
                 void* P, size_t p_bytes,
                 int B, int H, int n, int d, float scale, int causal, int dtype,
                 void* stream);

/* Naive backward: dQ, dK, dV from Q, K, V, the forward's O and P, and dO.
 * A pre-pass computes D_i = sum_c dO_ic O_ic into the workspace
 * (attn_workspace_bytes(B,H,n,d) bytes); dV = P^T dO and dS = P (dP - D)
 * then use the stored P. P and O must be attn_mat_fwd's outputs for the same
 * Q, K, V, scale and mask. */
int attn_mat_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const void* P, size_t p_bytes, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int n, int d, float scale, int causal, int dtype,
                 void* stream);

/* Naive forward then backward in one call (the forward also computes D from
 * dO, as attn_fwd_bwd does): same outputs as attn_fwd_bwd, plus P. */
int attn_mat_fwd_bwd(const void* Q, const void* K, const void* V, const void* dO,
                     void* O, float* L, void* P, size_t p_bytes,
                     void* dQ, void* dK, void* dV,
                     void* workspace, size_t workspace_bytes,
                     int B, int H, int n, int d, float scale, int causal, int dtype,
                     void* stream);

/* ---- Decode (Paper III) -------------------------------------------------
 * One decode step over a KV cache: for every sequence b the new token's key
 * and value are appended at row len_b of its cache head (when k_new/v_new are
 * given), and its query heads attend to the first T_b = len_b + 1 rows (len_b
 * without an append):
 *   O[b,h] = softmax_j(scale q[b,h] . K[b,g,j]) V[b,g,j],  g = h / (Hq/Hkv)
 *   L[b,h] = ln sum_j exp(scale q[b,h] . K[b,g,j])
 * Grouped-query attention: Hq query heads share Hkv cache heads (Hq a multiple
 * of Hkv; Hkv = 1 is multi-query attention). A step with no key writes O = 0
 * and L = -inf.
 *
 * Layout: q, O [B, Hq, d]; k_cache, v_cache [B, Hkv, n_cap, d] (row j of a
 * cache head is token j); k_new, v_new [B, Hkv, d]; L float32 [B, Hq] or NULL;
 * cache_lens: device int32 [B] (len_b, clamped to [0, n]) or NULL (every len_b
 * = n). n_cap >= n + 1 with an append, >= n without. bfloat16 only
 * (ATTN_E_UNSUPPORTED for float32). The caches are written only at row len_b.
 *
 * Work split: a workgroup owns one cache head, one split of its keys and up to
 * 32 of the query heads that read it, so each cache row is read once per
 * step; the keys are split (n + 1 rounded to 128-key tiles) until there are
 * about 512 workgroups, and a last pass merges the splits by log-sum-exp. The
 * merge needs attn_decode_workspace_bytes(...) bytes of 16-byte aligned
 * workspace (0 when the keys are not split; workspace may then be NULL). */
size_t attn_decode_workspace_bytes(int B, int Hq, int Hkv, int n, int d, int append);

int attn_decode(const void* q, const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                const int* cache_lens, void* O, float* L, void* workspace, size_t workspace_bytes,
                int B, int Hq, int Hkv, int n, int n_cap, int d, float scale, int dtype,
                void* stream);

/* Not an operation of the paper: error reporting of this interface.
 * Static, NUL-terminated description of a status code (never NULL). */
const char* attn_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_MI355X_H */
