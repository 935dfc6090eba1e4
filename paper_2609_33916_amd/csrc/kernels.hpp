// The three kernels of the fused attention forward+backward pass on gfx950.
//
//   fwd_kernel  (query-owner)  O, L and the backward's row vector D
//   dkdv_kernel (key-owner)    dK, dV; each workgroup owns a block of keys
//                              and sweeps the query tiles that see them
//   dq_kernel   (query-owner)  dQ; each workgroup owns a block of queries
//                              and sweeps the key tiles they see
//
// The scores S and probabilities P of a tile live only in registers: they
// are produced by one MFMA product and consumed as the operand of the next
// (the fused path of Fig. fig:concept, section sec:dnf-onf-machines). Each
// output element is written by exactly one lane and there are no atomics:
// dV and dK are accumulated by the workgroup that owns the key block (the
// per-key-column pass of Paper II, section sec:paper2-gv-fix) and dQ by the
// workgroup that owns the query block, with S and dP recomputed instead of
// persisting the score gradient (the persisted-gradient alternative costs an
// n^2 re-read, Paper II, section sec:paper2-gk-mechanism).
//
// Scores are handled in the base-2 domain: x = S_raw * sl2 with
// sl2 = |scale| * log2(e), P = 2^(x - m), and L is converted back to the
// natural log on output. A negative scale is folded into Q's sign.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace attn {

struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;   // optional: when set, D_i = sum_c dO_ic O_ic is written
  void* o;
  float* lse;
  float* dvec;    // optional: -D rows (with dout), D_i = sum_c dO_ic O_ic
  float* lse2;    // optional: base-2 log-sum-exp rows, log2 sum_j 2^(S_ij log2 e)
  long long head_stride;  // n * d elements
  int n;
  int ntiles;    // query tiles per head
  int nblocks;   // grid size
  float sl2;     // |scale| * log2(e), clamped away from 0
  uint32_t qflip;  // sign-bit mask applied to Q (negative scale)
  void* amat;      // materialising forward only: the attention matrix P
  long long lda;   // its row stride in elements (a multiple of 128)
};

struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  const float* lse2;   // base-2 log-sum-exp rows written by the forward
  const float* dvec;   // -D rows written by the forward (negated D)
  void* dq;
  void* dk;
  void* dv;
  long long head_stride;
  int n;
  int ntiles;
  int nblocks;
  float sl2;
  float dk_scale;  // scale (dK = s dS^T Q; K is read sign-flipped when scale < 0)
  float dq_scale;  // scale
  uint32_t qflip;
  const void* amat;  // materialising backward only: the stored P, read instead of recomputed
  long long lda;
  float* dqacc;      // atomic-dQ backward only: float32 [heads, n, d] accumulator (zeroed)
};

// ======================================================================
// Backward pre-pass (attn_bwd): -D_i = -sum_c dO_ic O_ic and the base-2 log-sum-
// exp L_i log2(e) for every row, from a stored O and L. HBM-bound: each row
// is read once as 16-byte chunks, a group of D/CH lanes per row reduces with
// cross-lane adds.
// ======================================================================
struct PrepArgs {
  const void* o;
  const void* dout;
  const float* lse;
  float* dvec;
  float* lse2;
  long long rows;   // B * H * n
};

template <typename T, int D>
__global__ void __launch_bounds__(256) bwd_prep_kernel(const PrepArgs a) {
  constexpr int CH = Elem<T>::CH;      // elements per 16-byte chunk
  constexpr int G = D / CH;            // lanes per row (4..32)
  constexpr int RPB = 256 / G;         // rows per block
  const int tid = threadIdx.x;
  const long long row = (long long)blockIdx.x * RPB + tid / G;
  const int part = tid % G;
  float acc = 0.f;
  if (row < a.rows) {
    const u32x4 x = *(const u32x4*)((const T*)a.o + row * D + part * CH);
    const u32x4 y = *(const u32x4*)((const T*)a.dout + row * D + part * CH);
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc += __uint_as_float(x[e] << 16) * __uint_as_float(y[e] << 16);
        acc += __uint_as_float(x[e] & 0xffff0000u) * __uint_as_float(y[e] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) acc += __uint_as_float(x[e]) * __uint_as_float(y[e]);
    }
  }
  // reduce over the G lanes of the row (G divides 64, groups are aligned)
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (row < a.rows && part == 0) {
    a.dvec[row] = -acc;   // stored negated: the backward kernels start dP from it
    if (a.lse) a.lse2[row] = a.lse[row] * kLog2e;
  }
}

// ======================================================================
// Forward: a workgroup owns BQ = 128 queries (32 per wave); K and V tiles of
// BKV = 64 keys are staged in LDS (double-buffered through registers).
// Per wave and key tile:  S^T = K Q^T (rows = keys, cols = the wave's 32
// queries), online softmax per column, O^T += V^T P^T.
// ======================================================================
template <typename T, int D, bool CAUSAL>
__global__ void __launch_bounds__(256, sizeof(T) == 2 ? 2 : 1) fwd_kernel(const FwdArgs a) {
  using E = Elem<T>;
  using Frag = typename E::frag;
  constexpr int BQ = 128, BKV = 64, NKB = BKV / 32, NDB = D / 32;
  static_assert(BKV == 64, "TransRead reads 64-row tiles");
  constexpr int KP = E::KP;
  constexpr int TD = D / (2 * KP);   // k-steps over d
  constexpr int T32 = 16 / KP;       // k-steps over a 32-row block
  // bf16 at d = 128: padded K/V tiles (Pad32)
  static constexpr bool P32 = sizeof(T) == 2 && D == 128;
  using TL = Tile<T, BKV, D, P32>;
  // two stages of (K, V) in distinct LDS objects: the loop is unrolled by
  // two so every access names its stage statically, which lets the compiler
  // see that reads of one stage never wait on the copy into the other
  __shared__ __attribute__((aligned(16))) T stA[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T stB[2][TL::ELEMS];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, c = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  int head, qt;
  block_map(blockIdx.x, a.nblocks, a.ntiles, CAUSAL, head, qt);
  const int n = a.n;
  const size_t hoff = (size_t)head * (size_t)a.head_stride;
  const T* Qg = (const T*)a.q + hoff;
  const T* Kg = (const T*)a.k + hoff;
  const T* Vg = (const T*)a.v + hoff;
  const int q0 = qt * BQ, qw0 = q0 + 32 * w, qi = qw0 + c;

  RowFrags<T, D> qf;
  qf.load(Qg, qi, n, h, a.qflip);

  const int kv_end = CAUSAL ? min(n, q0 + BQ) : n;
  const int nt = (kv_end + BKV - 1) / BKV;

  TileLoader<T, BKV, D, P32> kld(w, lane), vld(w, lane);
  kld.issue(stA[0], Kg, 0, n, w);
  vld.issue(stA[1], Vg, 0, n, w);
  kld.commit(stA[0]);
  vld.commit(stA[1]);
  __syncthreads();

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = zero16();
  float m_use = -INFINITY, lsum = 0.f;
  const float sl2 = a.sl2;

  auto step = [&](int it, T (&cur)[2][TL::ELEMS], T (&nxt)[2][TL::ELEMS]) __attribute__((always_inline)) {
    const int kv0 = it * BKV;
    if (it + 1 < nt) {
      kld.issue(nxt[0], Kg, kv0 + BKV, n, w);
      vld.issue(nxt[1], Vg, kv0 + BKV, n, w);
    }
    const bool active = !CAUSAL || kv0 <= qw0 + 31;
    if (active) {
      const T* kl = cur[0];
      const T* vl = cur[1];
      f32x16 s[NKB];
#pragma unroll
      for (int b = 0; b < NKB; ++b) {
        s[b] = zero16();
#pragma unroll
        for (int t = 0; t < TD; ++t) mma(s[b], RowRead<T, D, P32>::get(kl, b, t, h, c), qf.f[t]);
      }
      // bf16 at d = 128: K row reads six products ahead of the score products
      // (measured 1.5-2 % faster forward at n = 16384 than the compiler's two)
      if constexpr (sizeof(T) == 2 && D == 128) {
        ATTN_SCHED(kSchedDSRead, 6);
#pragma unroll
        for (int i = 0; i < NKB * TD; ++i) {
          ATTN_SCHED(kSchedMFMA, 1);
          ATTN_SCHED(kSchedDSRead, 1);
        }
      }
      // lane (h, c): s[b][j] = raw score of key kv0 + 32b + 16h + j, query qi
      const bool edge = (kv0 + BKV > n) || (CAUSAL && kv0 + BKV - 1 > qw0);
      if (edge) {
        // keys after `last` are masked; the lane's keys of block b are base_b + j
        const int last = CAUSAL ? min(qi, n - 1) : n - 1;
#pragma unroll
        for (int b = 0; b < NKB; ++b) {
          const int lim = last - (kv0 + 32 * b + 16 * h);
#pragma unroll
          for (int j = 0; j < 16; ++j) s[b][j] = (j > lim) ? -INFINITY : s[b][j];
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int b = 0; b < NKB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[b][j]);
      mx = halves_max(mx);
      const float mt = mx * sl2;
      const bool resc = mt > m_use + kRescaleThresh;
      if (__builtin_amdgcn_ballot_w64(resc)) {
        const float alpha = resc ? exp2_fast(m_use - mt) : 1.f;
        if (resc) m_use = mt;
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;
      }
      const float mb = (m_use == -INFINITY) ? 0.f : -m_use;
      float rs = 0.f;
#pragma unroll
      for (int b = 0; b < NKB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float p = exp2_fast(fmaf(s[b][j], sl2, mb));
          rs += p;
          s[b][j] = p;
        }
      lsum += rs;
      // the PV products at a raised wave priority (forward 1-3 % faster;
      // raising it for the score products and exponentials instead, as in
      // the backward kernels, measured 2.5 % slower)
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int b = 0; b < NKB; ++b)
#pragma unroll
        for (int t = 0; t < T32; ++t) {
          const Frag pf = FragFromAcc<T>::get(s[b], t);
#pragma unroll
          for (int db = 0; db < NDB; ++db)
            mma(oacc[db], TransRead<T, D, 64, P32>::get(vl, b, db, t, h, c), pf);
        }
      __builtin_amdgcn_s_setprio(0);
    }
    if (it + 1 < nt) {
      kld.commit(nxt[0]);
      vld.commit(nxt[1]);
    }
    __syncthreads();
  };
  for (int it = 0; it < nt; it += 2) {
    step(it, stA, stB);
    if (it + 1 < nt) step(it + 1, stB, stA);
  }

  // ---- epilogue: lane (h, c) holds O^T columns of query qi
  const float ltot = halves_sum(lsum);
  const float inv = 1.f / ltot;
  T* Og = (T*)a.o + hoff;
  const T* dOg = a.dout ? (const T*)a.dout + hoff : nullptr;
  float dpart = 0.f;
  if (qi < n) {
    // all dO loads before the first O store (the two may not be proven
    // disjoint, and a load after a store would wait for it)
    f32x4 g[NDB][4];
    if (dOg) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) g[db][q4] = Quad<T>::load(dOg + (size_t)qi * D + 32 * db + 8 * q4 + 4 * h);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int col = 32 * db + 8 * q4 + 4 * h;
        const float o0 = oacc[db][4 * q4 + 0] * inv, o1 = oacc[db][4 * q4 + 1] * inv;
        const float o2 = oacc[db][4 * q4 + 2] * inv, o3 = oacc[db][4 * q4 + 3] * inv;
        Quad<T>::store(Og + (size_t)qi * D + col, o0, o1, o2, o3);
        if (dOg) dpart += o0 * g[db][q4][0] + o1 * g[db][q4][1] + o2 * g[db][q4][2] + o3 * g[db][q4][3];
      }
  }
  const float dsum = halves_sum(dpart);
  if (qi < n && h == 0) {
    const size_t row = (size_t)head * n + qi;
    const float l2 = m_use + log2f(ltot);
    a.lse[row] = l2 * kLn2;
    if (dOg) {
      a.dvec[row] = -dsum;   // stored negated (the backward starts dP - D from it)
      a.lse2[row] = l2;
    }
  }
}

// ======================================================================
// Ping-pong forward (bf16): eight-wave workgroups of 256 queries in two
// groups of four waves. Waves w and w + 4 run on the same SIMD, one from
// each group, and a barrier after every phase keeps the groups half a key
// tile apart, so that on every SIMD one wave runs matrix products while the
// other runs the softmax arithmetic:
//   phase 2j:     group 0: G(j)       group 1: X(j - 1)
//   phase 2j + 1: group 0: X(j)       group 1: G(j)
// G(j) holds the score products of key tile j and the P V products of tile
// j - 1; X(j) the mask, row maximum, rescale and exponentials of tile j.
// Group 0 issues the copies of K(j + 1) and V(j) at the start of its G(j)
// and waits for them at the barrier after its X(j), two phases later;
// group 1 issues none. A tile slot is refilled only after the barrier that
// follows the last phase reading it. Wave w of group g = w / 4 owns the 32
// queries of block 2 (w % 4) + g, so the two waves of a SIMD see
// neighbouring query blocks and, under a causal mask, nearly the same keys.
// ======================================================================
// Tile copies of the ping-pong forward: the per-lane byte offsets of a full
// tile and of the one tile of the sequence that can end past row n - 1 (its
// rows >= n fetch row n - 1, as in TileLoader), so a copy costs one select
// per instruction instead of the clamp arithmetic.
template <int D, bool P> struct PpCopy {
  using L = TileLoader<bf16, 64, D, P>;
  static constexpr int NI = L::NI;
  unsigned off[NI], offr[NI];
  int rrow;   // first row of the tile that ends past row n - 1 (-1: none)
  __device__ __forceinline__ PpCopy(int w, int lane, int n) {
    const L ld(w, lane);
    rrow = (n % 64) ? n - n % 64 : -1;
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      if constexpr (P) {
        off[j] = ld.off[j];
        const int over = rrow + ld.xr[j] - (n - 1);
        offr[j] = (ld.off[j] != L::kSpare && over > 0) ? ld.off[j] - 2u * (unsigned)(over * D) : ld.off[j];
      } else {
        off[j] = 2u * (unsigned)ld.off[j];
        const int over = rrow + ld.xr[j] - (n - 1);
        offr[j] = over > 0 ? 2u * (unsigned)(ld.off[j] - over * D) : off[j];
      }
    }
  }
  __device__ __forceinline__ void issue(bf16* lds, const bf16* g, int row0, int w) const {
    const auto rs = dma_rsrc(g + (size_t)row0 * D);
    const bool rag = row0 == rrow;
#pragma unroll
    for (int j = 0; j < NI; ++j) dma16(rs, rag ? offr[j] : off[j], (ATTN_LDS void*)(lds + 512 * (w * NI + j)));
  }
};

__device__ __forceinline__ void phase_barrier() {
  // LDS reads complete (lgkmcnt(0)), no wait for outstanding tile copies
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

template <int D, bool CAUSAL>
__global__ void __launch_bounds__(512) fwd_pp_kernel(const FwdArgs a) {
  using T = bf16;
  constexpr int BQ = 256, BKV = 64, NKB = BKV / 32, NDB = D / 32, TD = D / 16, T32 = 2;
  // swizzled, unpadded K/V tiles: a tile copy moves 16 KB where the padded
  // 32-wide layout moves 20 KB (its spare chunks pass through the vector
  // memory path as well); the forward measured 1.2-1.6 % faster, with the
  // registers (218) to spare for the swizzle's per-lane offsets
  static constexpr bool P32 = false;
  using TL = Tile<T, BKV, D, P32>;
  // K and V slots in distinct LDS objects (loop unrolled by two), so that
  // reads of one slot never wait for a copy into the other
  __shared__ __attribute__((aligned(16))) T kA[TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T kB[TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T vA[TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T vB[TL::ELEMS];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, c = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = w >> 2, wi = w & 3;
  int head, qt;
  block_map(blockIdx.x, a.nblocks, a.ntiles, CAUSAL, head, qt);
  const int n = a.n;
  const size_t hoff = (size_t)head * (size_t)a.head_stride;
  const T* Qg = (const T*)a.q + hoff;
  const T* Kg = (const T*)a.k + hoff;
  const T* Vg = (const T*)a.v + hoff;
  const int q0 = qt * BQ, qw0 = q0 + 32 * (2 * wi + g), qi = qw0 + c;

  RowFrags<T, D> qf;
  qf.load(Qg, qi, n, h, a.qflip);

  const int kv_end = CAUSAL ? min(n, q0 + BQ) : n;
  const int nt = (kv_end + BKV - 1) / BKV;

  const PpCopy<D, P32> ld(wi, lane, n);
  if (g == 0) ld.issue(kA, Kg, 0, wi);
  __syncthreads();

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = zero16();
  f32x16 s[NKB];
  bf16x8 pf[NKB][T32];
  float m_use = -INFINITY, lsum = 0.f;
  const float sl2 = a.sl2;

  // G(j): scores of tile j (K in kc), then P V of tile j - 1 (V in vp).
  // Both run on every tile from j = 1 on: the phases are as long as their
  // slowest wave, so skipping a wave's products past its last key (causal)
  // or past the last tile saves no time, and there X(j) masks every key, so
  // P is zero and the extra P V adds zeros (every V slot holds finite rows
  // from j = 1 on).
  auto scores = [&](const T (&kc)[TL::ELEMS]) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < NKB; ++b) s[b] = zero16();
#pragma unroll
    for (int t = 0; t < TD; ++t)
#pragma unroll
      for (int b = 0; b < NKB; ++b) mma(s[b], RowRead<T, D, P32>::get(kc, b, t, h, c), qf.f[t]);
  };
  auto G = [&](const T (&kc)[TL::ELEMS], const T (&vp)[TL::ELEMS]) __attribute__((always_inline)) {
    scores(kc);
#pragma unroll
    for (int b = 0; b < NKB; ++b)
#pragma unroll
      for (int t = 0; t < T32; ++t)
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          mma(oacc[db], TransRead<T, D, 64, P32>::get(vp, b, db, t, h, c), pf[b][t]);
    // operand reads kept kAhead products ahead: the wave of the other group
    // on this SIMD is in its softmax phase and does not cover LDS latency
    constexpr int NS = NKB * TD, NP = NKB * T32 * NDB, kAhead = 6;
    ATTN_SCHED(kSchedDSRead, kAhead);
#pragma unroll
    for (int i = 0; i < NS + NP; ++i) {
      ATTN_SCHED(kSchedMFMA, 1);
      const int nx = i + kAhead;   // product whose operands are read next
      if (nx < NS) ATTN_SCHED(kSchedDSRead, 1);
      else if (nx < NS + NP) ATTN_SCHED(kSchedDSRead, 2);
    }
  };
  // X(j): softmax of tile j's scores into pf. Keys at or beyond n, and under
  // the causal mask keys after the query, are set to -inf by selection (the
  // scores of a slot never filled may be any bit pattern), so a tile with no
  // visible key gives P = 0 and leaves the row state unchanged.
  auto X = [&](int j) __attribute__((always_inline)) {
    __builtin_amdgcn_s_setprio(1);
    const int kv0 = j * BKV;
    // lane (h, c): s[b][k] = raw score of key kv0 + 32b + 16h + k, query qi
    const bool edge = (kv0 + BKV > n) || (CAUSAL && kv0 + BKV - 1 > qw0);
    if (edge) {
      const int last = CAUSAL ? min(qi, n - 1) : n - 1;
#pragma unroll
      for (int b = 0; b < NKB; ++b) {
        const int lim = last - (kv0 + 32 * b + 16 * h);
#pragma unroll
        for (int k = 0; k < 16; ++k) s[b][k] = (k > lim) ? -INFINITY : s[b][k];
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int b = 0; b < NKB; ++b)
#pragma unroll
      for (int k = 0; k < 16; ++k) mx = fmaxf(mx, s[b][k]);
    mx = halves_max(mx);
    const float mt = mx * sl2;
    const bool resc = mt > m_use + kRescaleThresh;
    if (__builtin_amdgcn_ballot_w64(resc)) {
      const float alpha = resc ? exp2_fast(m_use - mt) : 1.f;
      if (resc) m_use = mt;
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int k = 0; k < 16; ++k) oacc[db][k] *= alpha;
    }
    const float mb = (m_use == -INFINITY) ? 0.f : -m_use;
    float rs = 0.f;
#pragma unroll
    for (int b = 0; b < NKB; ++b) {
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const float p = exp2_fast(fmaf(s[b][k], sl2, mb));
        rs += p;
        s[b][k] = p;
      }
#pragma unroll
      for (int t = 0; t < T32; ++t) pf[b][t] = FragFromAcc<T>::get(s[b], t);
    }
    lsum += rs;
    __builtin_amdgcn_s_setprio(0);
  };
  // group 0 copies K(j + 1) into kn and V(j) into vc at the start of G(j)
  auto copies = [&](int j, T (&kn)[TL::ELEMS], T (&vc)[TL::ELEMS]) __attribute__((always_inline)) {
    if (g == 0) {
      if (j + 1 < nt) ld.issue(kn, Kg, (j + 1) * BKV, wi);
      if (j < nt) ld.issue(vc, Vg, j * BKV, wi);
    }
  };
  // key tile j >= 1: K(j) in kc, V(j - 1) in vp
  auto iter = [&](int j, T (&kc)[TL::ELEMS], T (&kn)[TL::ELEMS], T (&vp)[TL::ELEMS], T (&vc)[TL::ELEMS])
      __attribute__((always_inline)) {
    copies(j, kn, vc);
    G(kc, vp);
    phase_barrier();
    X(j);
    __syncthreads();
  };
  if (g == 1) phase_barrier();
  // tile 0: scores only
  copies(0, kB, vA);
  scores(kA);
  phase_barrier();
  X(0);
  __syncthreads();
  for (int j = 1; j <= nt; j += 2) {
    iter(j, kB, kA, vA, vB);
    if (j + 1 <= nt) iter(j + 1, kA, kB, vB, vA);
  }
  if (g == 0) phase_barrier();

  // ---- epilogue: lane (h, c) holds O^T columns of query qi
  const float ltot = halves_sum(lsum);
  const float inv = 1.f / ltot;
  T* Og = (T*)a.o + hoff;
  const T* dOg = a.dout ? (const T*)a.dout + hoff : nullptr;
  float dpart = 0.f;
  if (qi < n) {
    f32x4 gd[NDB][4];
    if (dOg) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) gd[db][q4] = Quad<T>::load(dOg + (size_t)qi * D + 32 * db + 8 * q4 + 4 * h);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int col = 32 * db + 8 * q4 + 4 * h;
        const float o0 = oacc[db][4 * q4 + 0] * inv, o1 = oacc[db][4 * q4 + 1] * inv;
        const float o2 = oacc[db][4 * q4 + 2] * inv, o3 = oacc[db][4 * q4 + 3] * inv;
        Quad<T>::store(Og + (size_t)qi * D + col, o0, o1, o2, o3);
        if (dOg) dpart += o0 * gd[db][q4][0] + o1 * gd[db][q4][1] + o2 * gd[db][q4][2] + o3 * gd[db][q4][3];
      }
  }
  const float dsum = halves_sum(dpart);
  if (qi < n && h == 0) {
    const size_t row = (size_t)head * n + qi;
    const float l2 = m_use + log2f(ltot);
    a.lse[row] = l2 * kLn2;
    if (dOg) {
      a.dvec[row] = -dsum;
      a.lse2[row] = l2;
    }
  }
}

// ======================================================================
// Materialising forward: the naive realisation in which the attention matrix
// is written to memory for the backward to read (Fig. fig:concept; the A
// array of Table tab:paper1-dram). Same tiling as fwd_kernel, two sweeps over
// the key tiles:
//   1. S^T = K Q^T for every tile, keeping each query's running maximum and
//      sum of 2^(S sl2 - max): the base-2 log-sum-exp L2 of the row;
//   2. S^T again, P = 2^(S sl2 - L2) (already normalised), P stored to row qi
//      of the matrix (input dtype, row stride lda, zeros where masked) and
//      O^T += V^T P^T.
// Each wave writes every key tile it visits in full (64 keys) for its 32
// queries; under the causal mask tiles that lie wholly after the wave's
// last query are neither visited nor written.
// ======================================================================
template <typename T, int D, bool CAUSAL>
__global__ void __launch_bounds__(256) mat_fwd_kernel(const FwdArgs a) {
  using E = Elem<T>;
  using Frag = typename E::frag;
  constexpr int BQ = 128, BKV = 64, NKB = BKV / 32, NDB = D / 32;
  static_assert(BKV == 64, "TransRead reads 64-row tiles");
  constexpr int KP = E::KP;
  constexpr int TD = D / (2 * KP);
  constexpr int T32 = 16 / KP;
  static constexpr bool P32 = sizeof(T) == 2 && D == 128;   // padded K/V tiles (Pad32)
  using TL = Tile<T, BKV, D, P32>;
  __shared__ __attribute__((aligned(16))) T stA[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T stB[2][TL::ELEMS];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, c = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  int head, qt;
  block_map(blockIdx.x, a.nblocks, a.ntiles, CAUSAL, head, qt);
  const int n = a.n;
  const size_t hoff = (size_t)head * (size_t)a.head_stride;
  const T* Qg = (const T*)a.q + hoff;
  const T* Kg = (const T*)a.k + hoff;
  const T* Vg = (const T*)a.v + hoff;
  const int q0 = qt * BQ, qw0 = q0 + 32 * w, qi = qw0 + c;
  T* Arow = (T*)a.amat + (size_t)head * n * a.lda + (size_t)qi * a.lda;

  RowFrags<T, D> qf;
  qf.load(Qg, qi, n, h, a.qflip);

  const int kv_end = CAUSAL ? min(n, q0 + BQ) : n;
  const int nt = (kv_end + BKV - 1) / BKV;
  const float sl2 = a.sl2;
  TileLoader<T, BKV, D, P32> kld(w, lane), vld(w, lane);

  // raw scores of key tile kv0 for this lane's query (masked to -inf)
  auto scores = [&](const T* kl, int kv0, f32x16 (&s)[NKB]) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < NKB; ++b) {
      s[b] = zero16();
#pragma unroll
      for (int t = 0; t < TD; ++t) mma(s[b], RowRead<T, D, P32>::get(kl, b, t, h, c), qf.f[t]);
    }
    const bool edge = (kv0 + BKV > n) || (CAUSAL && kv0 + BKV - 1 > qw0);
    if (edge) {
      const int last = CAUSAL ? min(qi, n - 1) : n - 1;
#pragma unroll
      for (int b = 0; b < NKB; ++b) {
        const int lim = last - (kv0 + 32 * b + 16 * h);
#pragma unroll
        for (int j = 0; j < 16; ++j) s[b][j] = (j > lim) ? -INFINITY : s[b][j];
      }
    }
  };

  // ---- sweep 1: row maximum and sum, K tiles only
  kld.issue(stA[0], Kg, 0, n, w);
  kld.commit(stA[0]);
  __syncthreads();
  float m_run = -INFINITY, lsum = 0.f;
  auto sweep1 = [&](int it, T (&cur)[2][TL::ELEMS], T (&nxt)[2][TL::ELEMS]) __attribute__((always_inline)) {
    const int kv0 = it * BKV;
    if (it + 1 < nt) kld.issue(nxt[0], Kg, kv0 + BKV, n, w);
    if (!CAUSAL || kv0 <= qw0 + 31) {
      f32x16 s[NKB];
      scores(cur[0], kv0, s);
      float mx = -INFINITY;
#pragma unroll
      for (int b = 0; b < NKB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[b][j]);
      const float mt = halves_max(mx) * sl2;
      if (mt > m_run) {
        lsum *= exp2_fast(m_run - mt);
        m_run = mt;
      }
      const float mb = (m_run == -INFINITY) ? 0.f : -m_run;
      float rs = 0.f;
#pragma unroll
      for (int b = 0; b < NKB; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) rs += exp2_fast(fmaf(s[b][j], sl2, mb));
      lsum += rs;
    }
    if (it + 1 < nt) kld.commit(nxt[0]);
    __syncthreads();
  };
  for (int it = 0; it < nt; it += 2) {
    sweep1(it, stA, stB);
    if (it + 1 < nt) sweep1(it + 1, stB, stA);
  }
  const float ltot = halves_sum(lsum);
  const float l2 = m_run + log2f(ltot);

  // ---- sweep 2: normalised P to memory and O = P V. A tile's P is kept
  // packed in registers and written at the top of the next step, next to the
  // next tile's LDS copies, so the waits for both overlap.
  kld.issue(stA[0], Kg, 0, n, w);
  vld.issue(stA[1], Vg, 0, n, w);
  kld.commit(stA[0]);
  vld.commit(stA[1]);
  __syncthreads();
  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = zero16();
  constexpr int NC = Run16<T>::NC;
  u32x4 pk[NKB][NC];
  int pk_col = -1;   // first key of the pending tile (wave-uniform), -1 if none
  auto flush = [&]() __attribute__((always_inline)) {
    if (pk_col >= 0 && qi < n) {
#pragma unroll
      for (int b = 0; b < NKB; ++b) store_run16<T>(Arow + pk_col + 32 * b + 16 * h, pk[b]);
    }
    pk_col = -1;
  };
  auto sweep2 = [&](int it, T (&cur)[2][TL::ELEMS], T (&nxt)[2][TL::ELEMS]) __attribute__((always_inline)) {
    const int kv0 = it * BKV;
    flush();
    if (it + 1 < nt) {
      kld.issue(nxt[0], Kg, kv0 + BKV, n, w);
      vld.issue(nxt[1], Vg, kv0 + BKV, n, w);
    }
    if (!CAUSAL || kv0 <= qw0 + 31) {
      f32x16 s[NKB];
      scores(cur[0], kv0, s);
#pragma unroll
      for (int b = 0; b < NKB; ++b) {
#pragma unroll
        for (int j = 0; j < 16; ++j) s[b][j] = exp2_fast(fmaf(s[b][j], sl2, -l2));
        Run16<T>::pack(s[b], pk[b]);
      }
      pk_col = kv0;
#pragma unroll
      for (int b = 0; b < NKB; ++b)
#pragma unroll
        for (int t = 0; t < T32; ++t) {
          Frag pf;
          if constexpr (sizeof(T) == 2) pf = __builtin_bit_cast(Frag, pk[b][t]);   // the stored values
          else pf = FragFromAcc<T>::get(s[b], t);
#pragma unroll
          for (int db = 0; db < NDB; ++db) mma(oacc[db], TransRead<T, D, 64, P32>::get(cur[1], b, db, t, h, c), pf);
        }
    }
    if (it + 1 < nt) {
      kld.commit(nxt[0]);
      vld.commit(nxt[1]);
    }
    __syncthreads();
  };
  for (int it = 0; it < nt; it += 2) {
    sweep2(it, stA, stB);
    if (it + 1 < nt) sweep2(it + 1, stB, stA);
  }
  flush();

  // ---- epilogue: O, L and (with dO) the backward's D and base-2 L rows
  T* Og = (T*)a.o + hoff;
  const T* dOg = a.dout ? (const T*)a.dout + hoff : nullptr;
  float dpart = 0.f;
  if (qi < n) {
    f32x4 g[NDB][4];   // dO loads first, as in fwd_kernel
    if (dOg) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) g[db][q4] = Quad<T>::load(dOg + (size_t)qi * D + 32 * db + 8 * q4 + 4 * h);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int col = 32 * db + 8 * q4 + 4 * h;
        const float o0 = oacc[db][4 * q4 + 0], o1 = oacc[db][4 * q4 + 1];
        const float o2 = oacc[db][4 * q4 + 2], o3 = oacc[db][4 * q4 + 3];
        Quad<T>::store(Og + (size_t)qi * D + col, o0, o1, o2, o3);
        if (dOg) dpart += o0 * g[db][q4][0] + o1 * g[db][q4][1] + o2 * g[db][q4][2] + o3 * g[db][q4][3];
      }
  }
  const float dsum = halves_sum(dpart);
  if (qi < n && h == 0) {
    const size_t row = (size_t)head * n + qi;
    a.lse[row] = l2 * kLn2;
    if (dOg) {
      a.dvec[row] = -dsum;   // stored negated (the backward starts dP - D from it)
      a.lse2[row] = l2;
    }
  }
}

// ======================================================================
// dK, dV: a workgroup owns BKV = 128 keys (32 per wave, held in registers as
// B operands); Q and dO tiles of BQ = 64 queries are staged in LDS with
// their base-2 log-sum-exp and D rows.
// Per wave and 32-query block:  S = Q K^T, dP = dO V^T  (rows = queries,
// cols = the wave's keys), P = 2^(S sl2 - L), dS = P (dP - D),
// dV^T += dO^T P, dK^T += Q^T dS.
// With MAT (materialising backward) S is not recomputed: each lane reads its
// column of P (16 query rows) straight from the stored matrix.
// ======================================================================
template <typename T, int D, bool CAUSAL, bool MAT = false>
__global__ void __launch_bounds__(256) dkdv_kernel(const BwdArgs a) {
  using E = Elem<T>;
  using Frag = typename E::frag;
  constexpr int BKV = 128, BQ = 64, NQB = BQ / 32, NDB = D / 32;
  static_assert(BQ == 64, "TransRead reads 64-row tiles");
  constexpr int KP = E::KP;
  constexpr int T32 = 16 / KP;
  using TL = Tile<T, BQ, D>;
  // two stages of (Q, dO) with their L and D rows, in distinct LDS objects
  // (loop unrolled by two, as in the forward)
  __shared__ __attribute__((aligned(16))) T stA[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T stB[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) float ldA[2][BQ];
  __shared__ __attribute__((aligned(16))) float ldB[2][BQ];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, c = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  int head, kt;
  block_map(blockIdx.x, a.nblocks, a.ntiles, false, head, kt);
  const int n = a.n;
  const size_t hoff = (size_t)head * (size_t)a.head_stride;
  const T* Qg = (const T*)a.q + hoff;
  const T* Kg = (const T*)a.k + hoff;
  const T* Vg = (const T*)a.v + hoff;
  const T* dOg = (const T*)a.dout + hoff;
  const float* Lg = a.lse2 + (size_t)head * n;
  const float* Dg = a.dvec + (size_t)head * n;
  const int k0 = kt * BKV, kw0 = k0 + 32 * w, kj = kw0 + c;

  // K is read sign-flipped for a negative scale (S = |s| Q (-K)^T), so the
  // Q tiles stay as stored and dK takes the signed scale
  RowFrags<T, D> kf, vf;
  if (!MAT) kf.load(Kg, kj, n, h, a.qflip);
  vf.load(Vg, kj, n, h, 0u);
  const T* Ag = MAT ? (const T*)a.amat + (size_t)head * n * a.lda : nullptr;

  const int q_begin = CAUSAL ? (k0 / BQ) * BQ : 0;
  const int nt = (n - q_begin + BQ - 1) / BQ;

  TileLoader<T, BQ, D> qld(w, lane), dold(w, lane);
  // base-2 LSE and D rows of the tile: one 4-byte-per-lane LDS DMA each
  // (waves 0 and 1); rows >= n fetch row n - 1 (masked by the kernel)
  auto load_rows = [&](int r0, T (&tl)[2][TL::ELEMS], float (&ld)[2][BQ]) __attribute__((always_inline)) {
    qld.issue(tl[0], Qg, r0, n, w);
    dold.issue(tl[1], dOg, r0, n, w);
    if (w < 2 && (!MAT || w == 1)) {   // MAT reads no L rows
      const int r = min(r0 + lane, n - 1);
      dma4(dma_rsrc(w == 0 ? Lg : Dg), 4u * (unsigned)r, (ATTN_LDS void*)(ld[w]));
    }
  };
  auto store_rows = [&](T (&tl)[2][TL::ELEMS]) __attribute__((always_inline)) {
    qld.commit(tl[0]);
    dold.commit(tl[1]);
  };
  load_rows(q_begin, stA, ldA);
  store_rows(stA);
  __syncthreads();

  f32x16 dk[NDB], dv[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) { dk[db] = zero16(); dv[db] = zero16(); }
  const float sl2 = a.sl2;

  auto step = [&](int it, T (&cur)[2][TL::ELEMS], float (&lcur)[2][BQ], T (&nxt)[2][TL::ELEMS],
                  float (&lnxt)[2][BQ]) __attribute__((always_inline)) {
    const int qt0 = q_begin + it * BQ;
    if (it + 1 < nt) load_rows(qt0 + BQ, nxt, lnxt);
    const T* ql = cur[0];
    const T* dol = cur[1];
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const int qb0 = qt0 + 32 * qb;
      if (CAUSAL && qb0 + 31 < kw0) continue;  // every query of the block precedes every key
      f32x16 s = zero16(), dp = zero16();
      if constexpr (MAT) {
        // lane (h, c): P of query qb0 + 16h + j, key kj (rows or keys >= n read as 0)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int q = qb0 + 16 * h + j;
          s[j] = (q < n && kj < n) ? (float)Ag[(size_t)q * a.lda + kj] : 0.f;
        }
      }
#pragma unroll
      for (int t = 0; t < D / (2 * KP); ++t) {
        if (!MAT) mma(s, RowRead<T, D>::get(ql, qb, t, h, c), kf.f[t]);
        mma(dp, RowRead<T, D>::get(dol, qb, t, h, c), vf.f[t]);
      }
      // lane (h, c): element j is query qb0 + 16h + j, key kj
      const f32x4* lp = (const f32x4*)&lcur[0][32 * qb + 16 * h];
      const f32x4* dp4 = (const f32x4*)&lcur[1][32 * qb + 16 * h];
      const bool edge = (qb0 + 31 >= n) || (CAUSAL && qb0 < kw0 + 31);
      // valid queries qb0 + 16h + j: lo <= j <= hi
      const int qbase = qb0 + 16 * h;
      const int lo = CAUSAL ? kj - qbase : -1, hi = n - 1 - qbase;
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        const f32x4 l4 = lp[j4], d4 = dp4[j4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = 4 * j4 + e;
          float p = MAT ? s[j] : exp2_fast(fmaf(s[j], sl2, -l4[e]));
          if (edge) p = (j < lo || j > hi) ? 0.f : p;
          s[j] = p;
          dp[j] = p * (dp[j] + d4[e]);   // d4 holds -D
        }
      }
#pragma unroll
      for (int t = 0; t < T32; ++t) {
        const Frag pf = FragFromAcc<T>::get(s, t);
        const Frag sf = FragFromAcc<T>::get(dp, t);
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          mma(dv[db], TransRead<T, D>::get(dol, qb, db, t, h, c), pf);
          mma(dk[db], TransRead<T, D>::get(ql, qb, db, t, h, c), sf);
        }
      }
    }
    if (it + 1 < nt) store_rows(nxt);
    __syncthreads();
  };
  for (int it = 0; it < nt; it += 2) {
    step(it, stA, ldA, stB, ldB);
    if (it + 1 < nt) step(it + 1, stB, ldB, stA, ldA);
  }

  if (kj < n) {
    T* dKg = (T*)a.dk + hoff;
    T* dVg = (T*)a.dv + hoff;
    const float sc = a.dk_scale;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int col = 32 * db + 8 * q4 + 4 * h;
        Quad<T>::store(dKg + (size_t)kj * D + col, dk[db][4 * q4] * sc, dk[db][4 * q4 + 1] * sc,
                       dk[db][4 * q4 + 2] * sc, dk[db][4 * q4 + 3] * sc);
        Quad<T>::store(dVg + (size_t)kj * D + col, dv[db][4 * q4], dv[db][4 * q4 + 1],
                       dv[db][4 * q4 + 2], dv[db][4 * q4 + 3]);
      }
  }
}

// ======================================================================
// dK, dV for bf16 on v_mfma_f32_16x16x32_bf16: a workgroup of NW waves owns
// 16 * KB * NW keys, KB blocks of 16 per wave (K and V rows of the wave's keys
// as B operands, dK^T and dV^T accumulators of 16 columns per block). Every
// Q / dO operand read from LDS feeds the KB blocks' products, so KB = 2
// halves the LDS bytes per product. V is held in registers; K too, except at
// d >= 64 (KL: KB = 2 at d = 128, KB = 3 at d = 64), where the K operands are
// read from an LDS copy of the workgroup's key block, staged once: in
// registers they would take VGPRs that two waves per SIMD do not leave (one
// wave's softmax VALU work overlaps the other's matrix products). At d = 128
// KL reads 0.625x the LDS bytes per product of 16-key waves. KB = 1 serves
// the atomic-dQ form and the materialising form at d = 32. Q and dO tiles of BQ queries (padded rows, Pad16; with their base-2
// LSE and -D rows) are staged in LDS;
// every 32 queries form one k step of the dV/dK products:
//   S = Q K^T, dP - D = dO V^T - D   (two 16-query blocks each; the dP
//                                     accumulators start from -D)
//   P = 2^(S sl2 - L), dS = P (dP - D)
//   dV^T += dO^T P, dK^T += Q^T dS  (contraction over the 32 queries)
// With MAT (the backward of the materialising path) S and the exponentials
// are not recomputed: the BQ x 16NW block of the stored P is staged in LDS
// next to Q and dO, and its transposed read is directly the P operand.
// With AQ (atomic dQ, the alternative to a separate dQ pass that recomputes
// S and dP) the workgroup also forms dQ = dS K for its keys: every wave writes
// its dS^T rows to an LDS tile [keys][queries] (double-buffered), and one
// step later each wave multiplies the whole tile by the workgroup's K block
// (kept in LDS) for a 16-column slice of d and adds the result to a float32
// accumulator in HBM with atomic adds (one per element and key block).
// ======================================================================
// (launch bound: at most 256 registers, so that two waves share each SIMD
// also when a workgroup has fewer than 8 waves)
template <int D, bool CAUSAL, int NW, int BQ, bool MAT = false, bool AQ = false, int KB = 1>
__global__ void __launch_bounds__(64 * NW, 2) dkdv16_kernel(const BwdArgs a) {
  constexpr int KW = 16 * KB;   // keys per wave: KB blocks of 16 share every Q / dO operand read
  constexpr int BKV = KW * NW, NPB = BQ / 32, TD = D / 32, NDB = D / 16;
  static_assert(!(MAT && AQ), "the materialising backward has its own dQ pass");
  static_assert(KB == 1 || !AQ, "the atomic-dQ form uses 16-key waves");
  constexpr int PT = MAT ? BQ * BKV : 8;
  constexpr int DST = AQ ? BKV * BQ : 8;   // dS^T tile [BKV keys][BQ queries]
  constexpr int KBL = AQ ? BKV * D : 8;    // the workgroup's K block [BKV][D]
  constexpr int TSZ = BQ * Pad16<D>::RS;  // a padded Q or dO tile (elements)
  __shared__ __attribute__((aligned(16))) bf16 stA[2][TSZ];
  __shared__ __attribute__((aligned(16))) bf16 stB[2][TSZ];
  __shared__ __attribute__((aligned(16))) float ldA[2][BQ];
  __shared__ __attribute__((aligned(16))) float ldB[2][BQ];
  __shared__ __attribute__((aligned(16))) bf16 ptA[PT];
  __shared__ __attribute__((aligned(16))) bf16 ptB[PT];
  __shared__ __attribute__((aligned(16))) bf16 dsA[DST];
  __shared__ __attribute__((aligned(16))) bf16 dsB[DST];
  __shared__ __attribute__((aligned(16))) bf16 kbl[KBL];
  constexpr bool KL = KB > 1 && D >= 64 && !MAT;
  static_assert(!KL || BQ == 32, "the KL step takes one pair block of queries");
  static_assert(KL || (BKV & (BKV - 1)) == 0, "the staged P block reads need a power-of-two key block");
  __shared__ __attribute__((aligned(16))) bf16 kst[KL ? BKV * Pad16<D>::RS : 8];

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, c = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  int head, kt;
  block_map(blockIdx.x, a.nblocks, a.ntiles, false, head, kt);
  const int n = a.n;
  const size_t hoff = (size_t)head * (size_t)a.head_stride;
  const bf16* Qg = (const bf16*)a.q + hoff;
  const bf16* Kg = (const bf16*)a.k + hoff;
  const bf16* Vg = (const bf16*)a.v + hoff;
  const bf16* dOg = (const bf16*)a.dout + hoff;
  const float* Lg = a.lse2 + (size_t)head * n;
  const float* Dg = a.dvec + (size_t)head * n;
  const int k0 = kt * BKV, kw0 = k0 + KW * w, kj = kw0 + c;
  const bf16* Ag = MAT ? (const bf16*)a.amat + (size_t)head * n * a.lda + k0 : nullptr;

  // B operands: row kj + 16 kb of K (sign-flipped for a negative scale; with
  // KL read from LDS instead) and of V; k-step t holds d in [32t + 8g, +8). K
  // is only needed to recompute S.
  bf16x8 kf[KB][TD], vf[KB][TD];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int t = 0; t < TD; ++t) {
      const int kr = kj + 16 * kb;
      u32x4 x = {0u, 0u, 0u, 0u}, y = {0u, 0u, 0u, 0u};
      if (kr < n) {
        if (!MAT && !KL) x = *(const u32x4*)(Kg + (size_t)kr * D + 32 * t + 8 * g);
        y = *(const u32x4*)(Vg + (size_t)kr * D + 32 * t + 8 * g);
      }
      x ^= (u32x4){a.qflip, a.qflip, a.qflip, a.qflip};
      kf[kb][t] = __builtin_bit_cast(bf16x8, x);
      vf[kb][t] = __builtin_bit_cast(bf16x8, y);
    }

  const int q_begin = CAUSAL ? (k0 / BQ) * BQ : 0;
  const int nt = (n - q_begin + BQ - 1) / BQ;

  TileLoader16P<BQ, D, NW> tld(w, lane);
  BlockLoader16<BQ, BKV, NW> pld(w, lane, MAT ? (int)a.lda : 0);
  auto load_rows = [&](int r0, bf16 (&tl)[2][TSZ], float (&lr)[2][BQ], bf16 (&pt)[PT])
      __attribute__((always_inline)) {
    tld.issue(tl[0], Qg, r0, n, w);
    tld.issue(tl[1], dOg, r0, n, w);
    if constexpr (MAT) pld.issue(pt, Ag, r0, n, w);
    if (w < 2 && (!MAT || w == 1)) {
      const int r = min(r0 + lane, n - 1);
      if (lane < BQ)
        dma4(dma_rsrc(w == 0 ? Lg : Dg), 4u * (unsigned)r, (ATTN_LDS void*)(lr[w]));
    }
  };
  load_rows(q_begin, stA, ldA, ptA);
  if constexpr (AQ) {
    TileLoader16<BKV, D, NW> kbld(w, lane);
    kbld.issue(kbl, Kg, k0, n, w);
  }
  if constexpr (KL) {
    TileLoader16P<BKV, D, NW> kld(w, lane);
    kld.issue(kst, Kg, k0, n, w);
  }
  __syncthreads();

  f32x4 dk[KB][NDB], dv[KB][NDB];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      dk[kb][db] = (f32x4){0.f, 0.f, 0.f, 0.f};
      dv[kb][db] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }
  // KL: a negative scale enters as the sign of sl2 instead of a sign flip of
  // K (the same products with the same signs)
  const float sl2 = (KL && a.qflip) ? -a.sl2 : a.sl2;

  // S (unless MAT) and dP - D of pair block pb (queries 32pb + [0, 32) of
  // the staged tile): the dP accumulators start from the staged row of -D
  // (lane group g's queries 4g + [0, 4) of each 16-query block), so the
  // product leaves dP - D without a subtraction per element. Every step form
  // does this the same way, so results do not depend on which form a tile
  // takes (and the atomic-dQ form's dK and dV equal the fused path's).
  auto sdp = [&](const bf16* ql, const bf16* dol, const float (&lr)[2][BQ], int pb, f32x4 (&sv)[KB][2],
                 f32x4 (&pv)[KB][2]) __attribute__((always_inline)) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const f32x4 init = *(const f32x4*)&lr[1][32 * pb + 16 * x + 4 * g];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        sv[kb][x] = (f32x4){0.f, 0.f, 0.f, 0.f};
        pv[kb][x] = init;
      }
    }
#pragma unroll
    for (int t = 0; t < TD; ++t) {
      bf16x8 kop[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) kop[kb] = KL ? row_read16p<D>(kst, KB * w + kb, t, g, c) : kf[kb][t];
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        if (!MAT) {
          const bf16x8 qa = row_read16p<D>(ql, 2 * pb + x, t, g, c);
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) mma16(sv[kb][x], qa, kop[kb]);
        }
        const bf16x8 oa = row_read16p<D>(dol, 2 * pb + x, t, g, c);
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) mma16(pv[kb][x], oa, vf[kb][t]);
      }
    }
  };
  // P = 2^(S sl2 - L) (MAT: P from the staged block, 16-key column block
  // kblk of the workgroup), dS = P (dP - D) as bf16 operands for the lane's
  // key `key` (pv holds dP - D); with MASK, queries >= n, keys >= n and
  // (causal) queries before the key get P = 0
  auto softmax = [&](const float (&lr)[2][BQ], const bf16* pt, int pb, int qp0, int key, int kblk, f32x4 (&sv)[2],
                     f32x4 (&pv)[2], bf16x8& pf, bf16x8& sf, auto mask) __attribute__((always_inline)) {
    constexpr bool M = decltype(mask)::value;
    bf16x8 praw;
    if constexpr (MAT) praw = tr_read16<BKV, BQ>(pt, 32 * pb, kblk, g, c);
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      f32x4 l4;
      if constexpr (!MAT) l4 = *(const f32x4*)&lr[0][32 * pb + 16 * x + 4 * g];
      // valid queries qbase + j: lo <= j <= hi (none for an absent key)
      const int qbase = qp0 + 16 * x + 4 * g;
      const int lo = CAUSAL ? key - qbase : -1;
      const int hi = ((MAT || AQ) && key >= n) ? -1 : n - 1 - qbase;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float p;
        if constexpr (MAT) p = (float)praw[4 * x + j];
        else p = exp2_fast(fmaf(sv[x][j], sl2, -l4[j]));
        if constexpr (M) p = (j < lo || j > hi) ? 0.f : p;
        sv[x][j] = p;
        pv[x][j] = p * pv[x][j];
      }
    }
    if constexpr (MAT && !M) pf = praw;
    else pf = frag16(sv[0], sv[1]);
    sf = frag16(pv[0], pv[1]);
  };
  // AQ: the wave's dS^T rows (keys kw0 + c) of pair block pb into the
  // [keys][queries] tile, 4 queries (8 bytes) per write
  auto put_ds = [&](bf16* dsT, int pb, const bf16x8& sf) __attribute__((always_inline)) {
    const int row = 16 * w + c;
    const u32x4 x = __builtin_bit_cast(u32x4, sf);
#pragma unroll
    for (int hx = 0; hx < 2; ++hx) {
      const int col = 32 * pb + 16 * hx + 4 * g;
      *(u32x2*)(dsT + row * BQ + 8 * ((col >> 3) ^ swz16<BQ>(row)) + (col & 7)) = (u32x2){x[2 * hx], x[2 * hx + 1]};
    }
  };
  // AQ: dQ of the queries of a finished step (dS^T in dsT) for this wave's
  // output tiles: d block w % (D/16), query blocks split between the waves
  // that share it; one float32 atomic add per element
  float* dQacc = AQ ? a.dqacc + (size_t)head * n * D : nullptr;
  auto dq_products = [&](const bf16* dsT, int qt0p) __attribute__((always_inline)) {
    if constexpr (AQ) {   // (not instantiated otherwise: its reads need power-of-two tiles)
      constexpr int NDT = D / 16, NQT = BQ / 16;
      constexpr int WPD = AQ ? NW / NDT : 1, QPW = NQT / WPD;
      static_assert(!AQ || (NW % NDT == 0 && NQT % WPD == 0), "dQ tiles must split evenly over the waves");
      const int dblk = w % NDT, qbase = (w / NDT) * QPW;
      // lane indexes made opaque here so that nothing of this phase is hoisted
      // out of the loop into registers that stay live across the other phases
      int gg = g, cc = c;
      asm volatile("" : "+v"(gg), "+v"(cc));
      bf16x8 kfr[BKV / 32];
  #pragma unroll
      for (int kb = 0; kb < BKV / 32; ++kb) kfr[kb] = tr_read16<D, BKV>(kbl, 32 * kb, dblk, gg, cc);
      // rows qt0p + 16 (qbase + i) + 4 gg + j of column 16 dblk + cc
      float* base = dQacc + (size_t)(qt0p + 16 * qbase + 4 * gg) * D + 16 * dblk + cc;
      const int qrow = qt0p + 16 * qbase + 4 * gg;
  #pragma unroll
      for (int i = 0; i < QPW; ++i) {
        f32x4 acc = (f32x4){0.f, 0.f, 0.f, 0.f};
  #pragma unroll
        for (int kb = 0; kb < BKV / 32; ++kb) mma16(acc, tr_read16<BQ, BKV>(dsT, 32 * kb, qbase + i, gg, cc), kfr[kb]);
  #pragma unroll
        for (int j = 0; j < 4; ++j)
          if (qrow + 16 * i + j < n) unsafeAtomicAdd(base + (16 * i + j) * D, acc[j]);
      }
    }
  };
  auto dvdk = [&](const bf16* ql, const bf16* dol, int pb, const bf16x8 (&pf)[KB], const bf16x8 (&sf)[KB])
      __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const bf16x8 oa = tr_read16p<D>(dol, 32 * pb, db, g, c);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) mma16(dv[kb][db], oa, pf[kb]);
      const bf16x8 qa = tr_read16p<D>(ql, 32 * pb, db, g, c);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) mma16(dk[kb][db], qa, sf[kb]);
    }
  };

  // AQ: dQ of the previous step, in a scheduling region of its own at the
  // top of a step (its dS^T tile was completed before the last barrier)
  auto dq_prev = [&](int it, const bf16* dprev) __attribute__((always_inline)) {
    if constexpr (AQ) {
      if (it > 0) {
        __builtin_amdgcn_sched_barrier(0);
        dq_products(dprev, q_begin + (it - 1) * BQ);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  // Pair blocks one after another; with MASK (tiles that touch the diagonal
  // or the end of the sequence) the masks are applied.
  auto step_seq = [&](int it, bf16 (&cur)[2][TSZ], float (&lcur)[2][BQ], bf16 (&pcur)[PT], bf16 (&dcur)[DST],
                      bf16 (&nxt)[2][TSZ], float (&lnxt)[2][BQ], bf16 (&pnxt)[PT], bf16 (&dprev)[DST], auto mask)
      __attribute__((always_inline)) {
    const int qt0 = q_begin + it * BQ;
    if (it + 1 < nt) load_rows(qt0 + BQ, nxt, lnxt, pnxt);
    dq_prev(it, dprev);
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      const int qp0 = qt0 + 32 * pb;
      if (CAUSAL && qp0 + 31 < kw0) {  // every query of the block precedes every key
        if constexpr (AQ) put_ds(dcur, pb, __builtin_bit_cast(bf16x8, (u32x4){0u, 0u, 0u, 0u}));
        continue;
      }
      f32x4 sv[KB][2], pv[KB][2];
      bf16x8 pf[KB], sf[KB];
      sdp(cur[0], cur[1], lcur, pb, sv, pv);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        softmax(lcur, pcur, pb, qp0, kj + 16 * kb, KB * w + kb, sv[kb], pv[kb], pf[kb], sf[kb], mask);
      if constexpr (AQ) put_ds(dcur, pb, sf[0]);
      dvdk(cur[0], cur[1], pb, pf, sf);
    }
    __syncthreads();
  };
  // KL steps (one pair block of 32 queries, every tile): one code path for
  // interior and masked tiles (two step forms measured about 400 bytes of
  // spills per lane). The exponentials of both key blocks, then one
  // wave-uniform branch around the mask selects (diagonal and last tiles),
  // with the first transposed reads of the dV/dK products issued before it.
  // Schedule: the S/dP products with their row reads eight ahead; the dV/dK
  // products with four transposed reads up front, then one per product.
  // Blocks whose queries all precede the wave's keys are computed and
  // masked (P = 0) rather than skipped: the diagonal tiles are a few of a
  // workgroup's.
  auto step_kl = [&](int it, bf16 (&cur)[2][TSZ], float (&lcur)[2][BQ], bf16 (&nxt)[2][TSZ], float (&lnxt)[2][BQ])
      __attribute__((always_inline)) {
    const int qt0 = q_begin + it * BQ;
    if (it + 1 < nt) load_rows(qt0 + BQ, nxt, lnxt, ptA);
    const bool need_mask = (CAUSAL && qt0 < k0 + BKV) || qt0 + BQ > n;
    // the S/dP products (at d = 64 also the exponentials) at a raised wave
    // priority: when both waves of a SIMD can issue, the one producing its
    // next P and dS goes first (dK/dV 1-3 % faster; at d = 128 another 2-5 %
    // with the exponentials back at the normal priority, which at d = 64
    // measured 8 % slower)
    __builtin_amdgcn_s_setprio(1);
    f32x4 sv[KB][2], pv[KB][2];
    sdp(cur[0], cur[1], lcur, 0, sv, pv);
    if constexpr (D > 64) __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const f32x4 l4 = *(const f32x4*)&lcur[0][16 * x + 4 * g];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) sv[kb][x][j] = exp2_fast(fmaf(sv[kb][x][j], sl2, -l4[j]));
    }
    __builtin_amdgcn_s_setprio(0);
    const bf16x8 oa0 = tr_read16p<D>(cur[1], 0, 0, g, c), qa0 = tr_read16p<D>(cur[0], 0, 0, g, c);
    ATTN_SCHED(kSchedDSRead, 8);
#pragma unroll
    for (int i = 0; i < 4 * TD * KB; ++i) {
      ATTN_SCHED(kSchedMFMA, 1);
      ATTN_SCHED(kSchedDSRead, 1);
    }
    if (need_mask) {
      // valid queries qbase + j: lo <= j <= hi
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int qbase = qt0 + 16 * x + 4 * g;
        const int hi = n - 1 - qbase;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int lo = CAUSAL ? kj + 16 * kb - qbase : -1;
#pragma unroll
          for (int j = 0; j < 4; ++j) sv[kb][x][j] = (j < lo || j > hi) ? 0.f : sv[kb][x][j];
        }
      }
    }
    bf16x8 pf[KB], sf[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int j = 0; j < 4; ++j) pv[kb][x][j] = sv[kb][x][j] * pv[kb][x][j];
      pf[kb] = frag16(sv[kb][0], sv[kb][1]);
      sf[kb] = frag16(pv[kb][0], pv[kb][1]);
    }
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const bf16x8 oa = db == 0 ? oa0 : tr_read16p<D>(cur[1], 0, db, g, c);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) mma16(dv[kb][db], oa, pf[kb]);
      const bf16x8 qa = db == 0 ? qa0 : tr_read16p<D>(cur[0], 0, db, g, c);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) mma16(dk[kb][db], qa, sf[kb]);
    }
    ATTN_SCHED(kSchedDSRead, 4);
#pragma unroll
    for (int i = 0; i < 2 * KB * NDB; ++i) {
      ATTN_SCHED(kSchedMFMA, 1);
      ATTN_SCHED(kSchedDSRead, 1);
    }
    __syncthreads();
  };
  // Interior tiles of the 16-key form at d = 128 (the atomic-dQ form; every
  // query sees every key of the workgroup, all rows valid): software-
  // pipelined, the S/dP products of pair block pb + 1 are issued next to the
  // exponentials of pair block pb, whose dV/dK products follow.
  auto step_inner = [&](int it, bf16 (&cur)[2][TSZ], float (&lcur)[2][BQ], bf16 (&pcur)[PT], bf16 (&dcur)[DST],
                        bf16 (&nxt)[2][TSZ], float (&lnxt)[2][BQ], bf16 (&pnxt)[PT], bf16 (&dprev)[DST])
      __attribute__((always_inline)) {
    const int qt0 = q_begin + it * BQ;
    if (it + 1 < nt) load_rows(qt0 + BQ, nxt, lnxt, pnxt);
    dq_prev(it, dprev);
    f32x4 sv[2][KB][2], pv[2][KB][2];
    sdp(cur[0], cur[1], lcur, 0, sv[0], pv[0]);
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      if (pb + 1 < NPB) sdp(cur[0], cur[1], lcur, pb + 1, sv[(pb + 1) & 1], pv[(pb + 1) & 1]);
      bf16x8 pf[KB], sf[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        softmax(lcur, pcur, pb, qt0 + 32 * pb, kj + 16 * kb, KB * w + kb, sv[pb & 1][kb], pv[pb & 1][kb], pf[kb],
                sf[kb], std::false_type{});
      if constexpr (AQ) put_ds(dcur, pb, sf[0]);
      dvdk(cur[0], cur[1], pb, pf, sf);
    }
    // schedule: S/dP of block 0 with its row reads running ahead; then per
    // block pb, its exponentials next to the next block's S/dP products and
    // next to its own dV/dK products (whose transposed reads run ahead). Two
    // reads and three VALU instructions per product slot while the next
    // block's S/dP products run: its row reads and the first transposed reads
    // of block pb (which the padded tiles leave the registers for), and the
    // exponentials of block pb spread over those products; four VALU
    // instructions per dV/dK product (the next block's exponentials).
    ATTN_SCHED(kSchedDSRead, 4);
#pragma unroll
    for (int i = 0; i < 4 * TD; ++i) { ATTN_SCHED(kSchedMFMA, 1); ATTN_SCHED(kSchedDSRead, 1); }
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
      if (pb + 1 < NPB) {
#pragma unroll
        for (int i = 0; i < 4 * TD; ++i) {
          ATTN_SCHED(kSchedMFMA, 1);
          ATTN_SCHED(kSchedDSRead, 2);
          ATTN_SCHED(kSchedVALU, 3);
        }
      }
#pragma unroll
      for (int i = 0; i < 2 * NDB; ++i) {
        ATTN_SCHED(kSchedMFMA, 1);
        ATTN_SCHED(kSchedDSRead, 2);
        ATTN_SCHED(kSchedVALU, 4);
      }
    }
    __syncthreads();
  };
  auto step = [&](int it, bf16 (&cur)[2][TSZ], float (&lcur)[2][BQ], bf16 (&pcur)[PT], bf16 (&dcur)[DST],
                  bf16 (&nxt)[2][TSZ], float (&lnxt)[2][BQ], bf16 (&pnxt)[PT], bf16 (&dprev)[DST])
      __attribute__((always_inline)) {
    const int qt0 = q_begin + it * BQ;
    const bool interior = qt0 + BQ <= n && (!CAUSAL || qt0 >= k0 + BKV - 1) &&
                          (!(MAT || AQ) || k0 + BKV <= n);
    // KL: one step form for every tile. The 16-key form at d = 128 pipelines
    // its interior tiles (at smaller d a pair block has too few products to
    // hide the exponentials behind)
    if constexpr (KL) {
      step_kl(it, cur, lcur, nxt, lnxt);
    } else if constexpr (D == 128 && !MAT && KB == 1) {
      if (interior) step_inner(it, cur, lcur, pcur, dcur, nxt, lnxt, pnxt, dprev);
      else step_seq(it, cur, lcur, pcur, dcur, nxt, lnxt, pnxt, dprev, std::true_type{});
    } else {
      // the materialising form with 32-key waves (d >= 64) takes the masked
      // step on every tile: a second step form spilled about 400 bytes per
      // lane at d = 128
      constexpr bool one_form = MAT && KB > 1 && D >= 64;
      if (interior && (MAT || KB > 1) && !one_form)
        step_seq(it, cur, lcur, pcur, dcur, nxt, lnxt, pnxt, dprev, std::false_type{});
      else
        step_seq(it, cur, lcur, pcur, dcur, nxt, lnxt, pnxt, dprev, std::true_type{});
    }
  };
  for (int it = 0; it < nt; it += 2) {
    step(it, stA, ldA, ptA, dsA, stB, ldB, ptB, dsB);
    if (it + 1 < nt) step(it + 1, stB, ldB, ptB, dsB, stA, ldA, ptA, dsA);
  }
  if constexpr (AQ) dq_products((nt - 1) & 1 ? dsB : dsA, q_begin + (nt - 1) * BQ);

#pragma unroll
  for (int kb = 0; kb < KB; ++kb) {
    const int kr = kj + 16 * kb;
    if (kr < n) {
      bf16* dKg = (bf16*)a.dk + hoff;
      bf16* dVg = (bf16*)a.dv + hoff;
      const float sc = a.dk_scale;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int col = 16 * db + 4 * g;
        Quad<bf16>::store(dKg + (size_t)kr * D + col, dk[kb][db][0] * sc, dk[kb][db][1] * sc, dk[kb][db][2] * sc,
                          dk[kb][db][3] * sc);
        Quad<bf16>::store(dVg + (size_t)kr * D + col, dv[kb][db][0], dv[kb][db][1], dv[kb][db][2], dv[kb][db][3]);
      }
    }
  }
}

// ======================================================================
// dQ: a workgroup owns BQ = 128 queries (32 per wave; Q and dO rows in
// registers as B operands, L and D per lane); K and V tiles of BKV = 64 keys
// are staged in LDS.
// Per wave and 32-key block:  S^T = K Q^T, dP^T = V dO^T (rows = keys,
// cols = the wave's queries), dS^T = P^T (dP^T - D), dQ^T += K^T dS^T.
// With MAT (materialising backward) S is not recomputed: the lane's 16 P
// values of a key block are 16 consecutive elements of its query's row of
// the stored matrix (bf16: loaded one key tile ahead into registers).
// ======================================================================
template <typename T, int D, bool CAUSAL, bool MAT = false>
__global__ void __launch_bounds__(256, sizeof(T) == 2 ? 2 : 1) dq_kernel(const BwdArgs a) {
  using E = Elem<T>;
  using Frag = typename E::frag;
  constexpr int BQ = 128, BKV = 64, NKB = BKV / 32, NDB = D / 32;
  static_assert(BKV == 64, "TransRead reads 64-row tiles");
  constexpr int KP = E::KP;
  constexpr int T32 = 16 / KP;
  // swizzled K/V tiles: the padded form (Pad32) frees 20 VGPRs here but measured
  // about 1 % slower at d = 128
  static constexpr bool P32 = false;
  using TL = Tile<T, BKV, D, P32>;
  // two stages of (K, V) in distinct LDS objects (loop unrolled by two)
  __shared__ __attribute__((aligned(16))) T stA[2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) T stB[2][TL::ELEMS];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, c = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  int head, qt;
  block_map(blockIdx.x, a.nblocks, a.ntiles, CAUSAL, head, qt);
  const int n = a.n;
  const size_t hoff = (size_t)head * (size_t)a.head_stride;
  const T* Qg = (const T*)a.q + hoff;
  const T* Kg = (const T*)a.k + hoff;
  const T* Vg = (const T*)a.v + hoff;
  const T* dOg = (const T*)a.dout + hoff;
  const int q0 = qt * BQ, qw0 = q0 + 32 * w, qi = qw0 + c;

  RowFrags<T, D> qf, of;
  if (!MAT) qf.load(Qg, qi, n, h, a.qflip);
  of.load(dOg, qi, n, h, 0u);
  const float lq = (!MAT && qi < n) ? a.lse2[(size_t)head * n + qi] : 0.f;
  const float dq_ = (qi < n) ? a.dvec[(size_t)head * n + qi] : 0.f;

  // stored P: 16-byte chunks of this lane's row, PC chunks per 16 elements
  constexpr int PC = sizeof(T), PCH = Elem<T>::CH;
  constexpr bool PREF = MAT && sizeof(T) == 2;   // float32: loaded at the top of the step
  const T* Arow = MAT ? (const T*)a.amat + (size_t)head * n * a.lda + (size_t)min(qi, n - 1) * a.lda : nullptr;
  auto pload = [&](int kv0, u32x4 (&r)[2][PC]) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < PC; ++e) r[kb][e] = *(const u32x4*)(Arow + kv0 + 32 * kb + 16 * h + PCH * e);
  };
  auto pget = [&](const u32x4 (&r)[PC], int j) __attribute__((always_inline)) -> float {
    if constexpr (sizeof(T) == 2) {
      const uint32_t x = r[j >> 3][(j & 7) >> 1];
      return __uint_as_float((j & 1) ? (x & 0xffff0000u) : (x << 16));
    } else {
      return __uint_as_float(r[j >> 2][j & 3]);
    }
  };

  const int kv_end = CAUSAL ? min(n, q0 + BQ) : n;
  const int nt = (kv_end + BKV - 1) / BKV;

  TileLoader<T, BKV, D, P32> kld(w, lane), vld(w, lane);
  kld.issue(stA[0], Kg, 0, n, w);
  vld.issue(stA[1], Vg, 0, n, w);
  kld.commit(stA[0]);
  vld.commit(stA[1]);
  __syncthreads();

  f32x16 dqa[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) dqa[db] = zero16();
  const float sl2 = a.sl2;

  u32x4 pA[2][PC], pB[2][PC];
  if constexpr (PREF) pload(0, pA);
  auto step = [&](int it, T (&cur)[2][TL::ELEMS], T (&nxt)[2][TL::ELEMS], u32x4 (&pc)[2][PC],
                  u32x4 (&pn)[2][PC]) __attribute__((always_inline)) {
    const int kv0 = it * BKV;
    if (it + 1 < nt) {
      kld.issue(nxt[0], Kg, kv0 + BKV, n, w);
      vld.issue(nxt[1], Vg, kv0 + BKV, n, w);
      if constexpr (PREF) pload(kv0 + BKV, pn);
    }
    if constexpr (MAT && !PREF) pload(kv0, pc);
    const T* kl = cur[0];
    const T* vl = cur[1];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      const int kb0 = kv0 + 32 * kb;
      if (CAUSAL && kb0 > qw0 + 31) continue;  // every key of the block follows every query
      // S, dP and dS at a raised wave priority, the dQ products at the normal
      // one: when both waves of a SIMD can issue, the one producing its next
      // dS goes first (dQ about 2 % faster at n = 16384 and at d = 64)
      __builtin_amdgcn_s_setprio(1);
      f32x16 s = zero16(), dp = zero16();
#pragma unroll
      for (int t = 0; t < D / (2 * KP); ++t) {
        if (!MAT) mma(s, RowRead<T, D, P32>::get(kl, kb, t, h, c), qf.f[t]);
        mma(dp, RowRead<T, D, P32>::get(vl, kb, t, h, c), of.f[t]);
      }
      // without the mask (bf16): keep the K / V row reads two ahead of the
      // S / dP products (measured 7 % faster at n = 2048, d = 128; under the
      // mask the same hint measured 5 % slower)
      if constexpr (!MAT && !CAUSAL && sizeof(T) == 2) {
        ATTN_SCHED(kSchedDSRead, 2);
#pragma unroll
        for (int i = 0; i < 2 * (D / (2 * KP)); ++i) {
          ATTN_SCHED(kSchedMFMA, 1);
          ATTN_SCHED(kSchedDSRead, 1);
        }
      }
      // lane (h, c): element j is key kb0 + 16h + j, query qi
      const bool edge = (kb0 + 31 >= n) || (CAUSAL && kb0 + 31 > qw0) || (MAT && qw0 + 31 >= n);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float p = MAT ? pget(pc[kb], j) : exp2_fast(fmaf(s[j], sl2, -lq));
        if (edge) {
          const int key = kb0 + 16 * h + j;
          if (key >= n || (CAUSAL && key > qi) || (MAT && qi >= n)) p = 0.f;
        }
        dp[j] = p * (dp[j] + dq_);   // dq_ holds -D
      }
      __builtin_amdgcn_s_setprio(0);
#pragma unroll
      for (int t = 0; t < T32; ++t) {
        const Frag sf = FragFromAcc<T>::get(dp, t);
#pragma unroll
        for (int db = 0; db < NDB; ++db) mma(dqa[db], TransRead<T, D, 64, P32>::get(kl, kb, db, t, h, c), sf);
      }
    }
    if (it + 1 < nt) {
      kld.commit(nxt[0]);
      vld.commit(nxt[1]);
    }
    __syncthreads();
  };
  for (int it = 0; it < nt; it += 2) {
    step(it, stA, stB, pA, pB);
    if (it + 1 < nt) step(it + 1, stB, stA, pB, pA);
  }

  if (qi < n) {
    T* dQg = (T*)a.dq + hoff;
    const float sc = a.dq_scale;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int col = 32 * db + 8 * q4 + 4 * h;
        Quad<T>::store(dQg + (size_t)qi * D + col, dqa[db][4 * q4] * sc, dqa[db][4 * q4 + 1] * sc,
                       dqa[db][4 * q4 + 2] * sc, dqa[db][4 * q4 + 3] * sc);
      }
  }
}

// ======================================================================
// Decode (Paper III): one new query token per head against a KV cache.
//
// decode_append_kernel writes the new token's key and value at row len_b of
// its cache head. decode_kernel then covers keys [0, T_b) of every cache head
// (T_b = len_b + 1 with an append): a workgroup owns one cache head, one
// split of the keys (``chunk`` keys, a multiple of 128) and up to 32 of the
// query heads that share the cache head (GQA; MQA when there is one cache
// head), so K and V are read once for the whole group. The group's queries
// are the 32 columns of S^T = K Q^T (missing heads are zero columns); each
// wave takes one 32-key block of every 128-key tile with its own online
// softmax (base 2), the waves' partial (max, sum, O) are merged through LDS
// at the end, and with several splits decode_combine_kernel merges the
// splits by their log-sum-exp.
// ======================================================================
struct DecArgs {
  const void* q;        // [B, Hq, d]
  const void* kc;       // [B, Hkv, n_cap, d]
  const void* vc;
  const void* k_new;    // [B, Hkv, d] or null
  const void* v_new;
  const int* lens;      // [B] tokens cached before the step, or null (all n)
  float* part;          // splits > 1: [B*Hq][nsplit][d] unnormalised O, then [B*Hq][nsplit] (max2, sum)
  void* o;              // [B, Hq, d]
  float* lse;           // [B, Hq] natural log, or null
  int rows;            // B * Hq
  int Hq, Hkv, G, n, n_cap, append;
  int fuse_append;     // decode_kernel writes the new row itself (one query chunk per cache head)
  int chunk, nsplit, qchunks;
  float sl2;
  uint32_t qflip;
};

__device__ __forceinline__ int dec_len(const DecArgs& a, int b) {
  const int len = a.lens ? a.lens[b] : a.n;
  return min(max(len, 0), a.n);     // lengths are clamped to [0, n]
}

template <typename T, int D>
__global__ void __launch_bounds__(256) decode_append_kernel(const DecArgs a, int B) {
  constexpr int CH = Elem<T>::CH, CPR = D / CH;     // 16-byte chunks per row
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long rows = (long long)B * a.Hkv;
  if (i >= 2 * rows * CPR) return;
  const int which = (int)(i / (rows * CPR));         // 0: key, 1: value
  const long long r = (i / CPR) % rows;              // b * Hkv + hk
  const int ch = (int)(i % CPR);
  const int b = (int)(r / a.Hkv);
  const int pos = dec_len(a, b);
  const T* src = (const T*)(which ? a.v_new : a.k_new) + r * D + ch * CH;
  T* dst = (T*)(which ? a.vc : a.kc) + (r * a.n_cap + pos) * D + ch * CH;
  *(u32x4*)dst = *(const u32x4*)src;
}

template <int D>
__global__ void __launch_bounds__(256) decode_kernel(const DecArgs a) {
  using T = bf16;
  using E = Elem<T>;
  using Frag = typename E::frag;
  constexpr int BKV = 64, NKB = 2, NDB = D / 32;
  constexpr int KP = E::KP, TD = D / (2 * KP), T32 = 16 / KP;
  using TL = Tile<T, BKV, D>;
  static_assert(BKV == 64, "TransRead reads 64-row tiles");
  // V only, two stages of [rows 0-63, rows 64-127]; K goes straight to
  // registers (the score product reads K rows as they are stored)
  __shared__ __attribute__((aligned(16))) T st[2][2][TL::ELEMS];
  __shared__ __attribute__((aligned(16))) float mlw[2][4][32];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, c = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int split = blockIdx.x;
  const int grp = blockIdx.y;                        // (b, hk, qc)
  const int qc = grp % a.qchunks;
  const int bh = grp / a.qchunks;                    // b * Hkv + hk
  const int b = bh / a.Hkv, hk = bh % a.Hkv;
  const int T_b = dec_len(a, b) + a.append;
  const int k_lo = split * a.chunk, k_hi = min(T_b, k_lo + a.chunk);
  const int h0 = hk * a.G + qc * 32;                 // first query head of this workgroup
  const int nq = min(32, a.G - qc * 32);             // query heads in it
  const size_t kvoff = (size_t)bh * a.n_cap * D;
  const T* Kg = (const T*)a.kc + kvoff;
  const T* Vg = (const T*)a.vc + kvoff;
  const T* Qg = (const T*)a.q + ((size_t)b * a.Hq + h0) * D;

  RowFrags<T, D> qf;
  qf.load(Qg, c, nq, h, a.qflip);
  const float sl2 = a.sl2;
  const int sub = w >> 1, kb = w & 1;                // this wave: sub-tile and 32-key block
  const int nt = k_hi > k_lo ? (k_hi - k_lo + 127) / 128 : 0;

  TileLoader<T, BKV, D> ld(w, lane);
  // this wave's 32 K rows of a step as A operands: lane c takes key
  // kv0 + 32w + perm32(c), k-step t its columns 16t + 8h (the layout a row
  // read of a permuted LDS tile would give); rows past the split repeat its
  // last row (their scores are masked)
  auto kload = [&](int kv0, u32x4 (&kr)[TD]) __attribute__((always_inline)) {
    const int row = min(kv0 + 32 * w + perm32(c), k_hi - 1);
    const T* src = Kg + (size_t)row * D + 8 * h;
#pragma unroll
    for (int t = 0; t < TD; ++t) kr[t] = *(const u32x4*)(src + 16 * t);
  };
  auto issue = [&](T (&stg)[2][TL::ELEMS], u32x4 (&kr)[TD], int kv0) __attribute__((always_inline)) {
    ld.issue(stg[0], Vg, kv0, k_hi, w);
    ld.issue(stg[1], Vg, kv0 + 64, k_hi, w);
    kload(kv0, kr);
  };
  // the workgroup whose split holds row len_b writes the new key and value
  // there before any of its copies reads the row (no other workgroup reads it)
  if (a.fuse_append) {
    const int pos = T_b - 1;
    if (pos >= k_lo && pos < k_hi) {
      constexpr int CPR = D / 8;
      if (tid < 2 * CPR) {
        const int which = tid / CPR, ch = tid % CPR;
        const T* src = (const T*)(which ? a.v_new : a.k_new) + (size_t)bh * D + 8 * ch;
        T* dst = (T*)(which ? a.vc : a.kc) + kvoff + (size_t)pos * D + 8 * ch;
        *(u32x4*)dst = *(const u32x4*)src;
        __threadfence();
      }
      __syncthreads();
    }
  }
  u32x4 kA[TD], kB[TD];
  if (nt > 0) issue(st[0], kA, k_lo);
  __syncthreads();

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = zero16();
  float m_use = -INFINITY, lsum = 0.f;

  auto step = [&](int it, T (&cur)[2][TL::ELEMS], u32x4 (&kcur)[TD], T (&nxt)[2][TL::ELEMS],
                  u32x4 (&knxt)[TD]) __attribute__((always_inline)) {
    const int kv0 = k_lo + it * 128;
    if (it + 1 < nt) issue(nxt, knxt, kv0 + 128);
    const int kb0 = kv0 + 64 * sub + 32 * kb;        // first key of this wave's block (= kv0 + 32w)
    if (kb0 < k_hi) {
      const T* vl = cur[sub];
      f32x16 s = zero16();
#pragma unroll
      for (int t = 0; t < TD; ++t) mma(s, __builtin_bit_cast(Frag, kcur[t]), qf.f[t]);
      // lane (h, c): s[j] = raw score of key kb0 + 16h + j for query column c
      if (kb0 + 32 > k_hi) {
        const int lim = k_hi - 1 - (kb0 + 16 * h);
#pragma unroll
        for (int j = 0; j < 16; ++j) s[j] = (j > lim) ? -INFINITY : s[j];
      }
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[j]);
      const float mt = halves_max(mx) * sl2;
      const bool resc = mt > m_use + kRescaleThresh;
      if (__builtin_amdgcn_ballot_w64(resc)) {
        const float alpha = resc ? exp2_fast(m_use - mt) : 1.f;
        if (resc) m_use = mt;
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;
      }
      const float mb = (m_use == -INFINITY) ? 0.f : -m_use;
      float rs = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = exp2_fast(fmaf(s[j], sl2, mb));
        rs += p;
        s[j] = p;
      }
      lsum += rs;
#pragma unroll
      for (int t = 0; t < T32; ++t) {
        const Frag pf = FragFromAcc<T>::get(s, t);
#pragma unroll
        for (int db = 0; db < NDB; ++db) mma(oacc[db], TransRead<T, D>::get(vl, kb, db, t, h, c), pf);
      }
    }
    __syncthreads();
  };
  for (int it = 0; it < nt; it += 2) {
    step(it, st[0], kA, st[1], kB);
    if (it + 1 < nt) step(it + 1, st[1], kB, st[0], kA);
  }

  // ---- merge the four waves through LDS (the stage memory is free now):
  // O parts [4][D][32] over both stages, maxima and sums [4][32] each
  float* ow = (float*)&st[0][0][0];
  float* mw = &mlw[0][0][0];
  float* lw = &mlw[1][0][0];
  static_assert(4 * D * 32 * 4 <= 2 * 2 * TL::ELEMS * 2, "merge buffer exceeds the stages");
  const float ltot = halves_sum(lsum);
  if (h == 0) {
    mw[w * 32 + c] = m_use;
    lw[w * 32 + c] = ltot;
  }
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int dd = 32 * db + 8 * (j >> 2) + 4 * h + (j & 3);
      ow[(w * D + dd) * 32 + c] = oacc[db][j];
    }
  __syncthreads();
  // thread -> query column qq and D/8 consecutive d values
  const int qq = tid & 31, dpart = tid >> 5;
  constexpr int DPT = D / 8;
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < 4; ++v) M = fmaxf(M, mw[v * 32 + qq]);
  float f[4], l = 0.f;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    f[v] = (M == -INFINITY) ? 0.f : exp2_fast(mw[v * 32 + qq] - M);
    l += f[v] * lw[v * 32 + qq];
  }
  if (qq < nq) {
    const size_t row = (size_t)b * a.Hq + h0 + qq;
    float r[DPT];
#pragma unroll
    for (int e = 0; e < DPT; ++e) {
      const int dd = dpart * DPT + e;
      float acc = 0.f;
#pragma unroll
      for (int v = 0; v < 4; ++v) acc += f[v] * ow[(v * D + dd) * 32 + qq];
      r[e] = acc;
    }
    if (a.nsplit == 1) {
      const float inv = l > 0.f ? 1.f / l : 0.f;
      T* Og = (T*)a.o + row * D + dpart * DPT;
#pragma unroll
      for (int e4 = 0; e4 < DPT / 4; ++e4)
        Quad<T>::store(Og + 4 * e4, r[4 * e4] * inv, r[4 * e4 + 1] * inv, r[4 * e4 + 2] * inv, r[4 * e4 + 3] * inv);
      if (a.lse && dpart == 0) a.lse[row] = l > 0.f ? (M + log2f(l)) * kLn2 : -INFINITY;
    } else {
      // partials: [rows][nsplit][D] unnormalised O, then [rows][nsplit] (max2, sum)
      float* pml = a.part + (size_t)a.rows * a.nsplit * D + (row * a.nsplit + split) * 2;
      if (dpart == 0) {
        pml[0] = M;
        pml[1] = l;
      }
      float* po = a.part + (row * a.nsplit + split) * D + dpart * DPT;
#pragma unroll
      for (int e4 = 0; e4 < DPT / 4; ++e4)
        *(f32x4*)(po + 4 * e4) = (f32x4){r[4 * e4], r[4 * e4 + 1], r[4 * e4 + 2], r[4 * e4 + 3]};
    }
  }
}

// Merge the splits of decode_kernel: per (b, query head), O = sum_s 2^(m_s - M)
// O_s / sum_s 2^(m_s - M) l_s and L = (M + log2 l) ln 2. One workgroup per
// row: thread t takes 4 consecutive d values (t % (D/4)) of the splits
// s = t / (D/4) + k * SL, and the SL partial sums are added through LDS.
template <typename T, int D>
__global__ void __launch_bounds__(256) decode_combine_kernel(const float* part, void* o, float* lse, int rows,
                                                             int nsplit) {
  // one workgroup per query row; thread t takes 4 of the d values (dl) of
  // the splits sl, sl + SL, ...; it folds them into its own running
  // (max, sum, O) with the log-sum-exp rule, U splits per pass with all
  // their loads issued before the first fold, and the SL partial states of
  // each dl are folded together through LDS at the end
  constexpr int DL = D / 4, SL = 256 / DL, U = 8;
  __shared__ float smax[SL][DL], ssum[SL][DL];
  __shared__ __attribute__((aligned(16))) f32x4 sacc[SL][DL];
  const int row = blockIdx.x, t = threadIdx.x, dl = t % DL, sl = t / DL;
  const float* po = part + (size_t)row * nsplit * D + 4 * dl;
  const f32x2* pml = (const f32x2*)(part + (size_t)rows * nsplit * D + (size_t)row * nsplit * 2);
  float mt = -INFINITY, lt = 0.f;
  f32x4 acc = (f32x4){0.f, 0.f, 0.f, 0.f};
  // fold one partial state (m: base-2 max, l: sum, v: unnormalised O) into (mt, lt, acc)
  auto fold = [&](float m, float l, f32x4 v) __attribute__((always_inline)) {
    if (m == -INFINITY) return;   // an empty split
    const float nm = fmaxf(mt, m);
    const float a = (mt == -INFINITY) ? 0.f : exp2_fast(mt - nm), b = exp2_fast(m - nm);
    lt = lt * a + l * b;
    acc = acc * a + v * b;
    mt = nm;
  };
  for (int s0 = sl; s0 < nsplit; s0 += SL * U) {
    f32x2 ml[U];
    f32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + SL * u;
      ml[u] = (f32x2){-INFINITY, 0.f};
      v[u] = (f32x4){0.f, 0.f, 0.f, 0.f};
      if (s < nsplit) {
        ml[u] = pml[s];
        v[u] = *(const f32x4*)(po + (size_t)s * D);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) fold(ml[u][0], ml[u][1], v[u]);
  }
  smax[sl][dl] = mt;
  ssum[sl][dl] = lt;
  sacc[sl][dl] = acc;
  __syncthreads();
  if (t < DL) {
    mt = -INFINITY;
    lt = 0.f;
    acc = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < SL; ++k) fold(smax[k][t], ssum[k][t], sacc[k][t]);
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    Quad<T>::store((T*)o + (size_t)row * D + 4 * t, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    if (lse && t == 0) lse[row] = lt > 0.f ? (mt + log2f(lt)) * kLn2 : -INFINITY;
  }
}

// ======================================================================
// Atomic-dQ support: zero the float32 accumulator, then dQ = scale * acc in
// the output dtype. HBM-bound, 8 elements per thread.
// ======================================================================
static __global__ void __launch_bounds__(256) zero_f32_kernel(float* p, long long n8) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n8) {
    ((f32x4*)p)[2 * i] = (f32x4){0.f, 0.f, 0.f, 0.f};
    ((f32x4*)p)[2 * i + 1] = (f32x4){0.f, 0.f, 0.f, 0.f};
  }
}

template <typename T>
__global__ void __launch_bounds__(256) dq_finalize_kernel(const float* acc, T* dq, long long n8, float scale) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n8) {
    const f32x4 x = ((const f32x4*)acc)[2 * i], y = ((const f32x4*)acc)[2 * i + 1];
    Quad<T>::store(dq + 8 * i, x[0] * scale, x[1] * scale, x[2] * scale, x[3] * scale);
    Quad<T>::store(dq + 8 * i + 4, y[0] * scale, y[1] * scale, y[2] * scale, y[3] * scale);
  }
}

}  // namespace attn
