// Device building blocks for the gfx950 attention kernels: element traits,
// matrix-core (MFMA) wrappers, LDS tile layout and operand reads, lane-half
// reductions and the workgroup -> (head, tile) schedule.
//
// MFMA 32x32 register layouts (wave64, lane l, half h = l / 32, c = l % 32):
//   A operand   : row c, k slots [h*KP, h*KP + KP)
//   B operand   : col c, same k slots
//   accumulator : col c, row R(h, j) = 8*(j/4) + 4*h + (j%4), j in [0, 16)
// with KP = 8 for v_mfma_f32_32x32x16_bf16 and KP = 1 for
// v_mfma_f32_32x32x2_f32. Only the accumulator layout matters for
// correctness: any order of k slots works as long as A and B agree.
//
// Tiles in LDS are row-major (contiguous along d) and the rows of every
// 32-row block are stored permuted (srow below) so that
//  * a "row read" (A operand = tile rows, contraction over d) has lane c read
//    stored row c, and its accumulator row R(h, j) is logical row 16h + j;
//    lane half h then owns 16 consecutive logical rows, which is exactly the
//    k-slot order the next product needs when the accumulator is reused as
//    an operand (P and dS are never written to memory);
//  * a "transposed read" (A operand = tile columns, contraction over rows)
//    gets 8 consecutive logical rows per lane: for bf16 with two
//    ds_read_b64_tr_b16 (4 rows x 16 columns per 16-lane group), for float32
//    with one 4-byte read per MFMA.
// bf16 rows are unpadded and their 16-byte chunks XOR-swizzled (swz): LDS
// has 64 four-byte banks (16 slots of 16 bytes per 256-byte line); each
// ds_read_b128 pass serves 16 lanes and each ds_read_b64(_tr_b16) pass a
// half-wave, and a pass is conflict-free when its lanes touch distinct
// slots (see swz16 for which lanes share a pass). swz makes the rows of a
// row read and the 4 rows x 4 chunks of a transposed read land on distinct
// slots. Two padded forms trade LDS for addresses that are a lane base plus
// an immediate offset: Pad32 (the forward's K/V tiles at d = 128) and Pad16
// (the Q/dO tiles of the 16-wide dK/dV kernel).
// float32 rows are padded by one element instead.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define ATTN_LDS __attribute__((address_space(3)))

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// The running row maximum used for the exponentials is only moved when the
// true maximum exceeds it by more than this many powers of two; exponentials
// then stay below 2^8 and most key tiles skip rescaling the accumulators.
constexpr float kRescaleThresh = 8.0f;

// ---------------------------------------------------------------- traits --
template <typename T> struct Elem;
template <> struct Elem<bf16> {
  using frag = bf16x8;               // one MFMA operand per lane
  static constexpr int KP = 8;       // k slots per lane per MFMA
  static constexpr int PAD = 0;      // rows unpadded, chunks swizzled
  static constexpr int CH = 8;       // elements per 16-byte chunk
};
template <> struct Elem<float> {
  using frag = float;
  static constexpr int KP = 1;
  static constexpr int PAD = 1;
  static constexpr int CH = 4;
};

// ----------------------------------------------------- schedule hints --
// Instruction classes for __builtin_amdgcn_sched_group_barrier: the
// pipelined loops ask the scheduler to alternate matrix products with the
// LDS reads that feed later products and with independent VALU work.
enum : int { kSchedVALU = 0x2, kSchedMFMA = 0x8, kSchedDSRead = 0x100 };
#define ATTN_SCHED(mask, count) __builtin_amdgcn_sched_group_barrier((mask), (count), 0)

// ------------------------------------------------------------------ MFMA --
__device__ __forceinline__ void mma(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x16& acc, float a, float b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int j = 0; j < 16; ++j) z[j] = 0.f;
  return z;
}

// ------------------------------------------------------- permuted rows --
// perm32(r): logical row held by accumulator row r once operand rows are
// read through srow; perm32_inv is its inverse.
__host__ __device__ constexpr int perm32(int r) { return ((r >> 2) & 1) * 16 + (r >> 3) * 4 + (r & 3); }
__host__ __device__ constexpr int perm32_inv(int x) { return ((x >> 2) & 3) * 8 + (x >> 4) * 4 + (x & 3); }
// stored row of logical row x (permutation inside each 32-row block)
__host__ __device__ constexpr int srow(int x) { return (x & ~31) | perm32_inv(x & 31); }

// 16-byte chunk swizzle of stored row s of a bf16 tile with D columns
// (D/8 chunks per row, 16/(D/8) rows per 256-byte bank line).
template <int D> __host__ __device__ constexpr int swz(int s) {
  return D == 128 ? 4 * (s & 3) + ((s >> 2) & 3)
       : D == 64  ? 4 * ((s >> 1) & 1) + ((s >> 2) & 3)
                  : ((s >> 2) & 3);
}

// ------------------------------------------------------ lane-half ops --
// Lanes c and c + 32 hold the two halves of the same accumulator column.
__device__ __forceinline__ float halves_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float halves_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------- conversions --
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16 a = (bf16)lo, b = (bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Operand fragment for k-step t from 16 accumulator values that are already
// in the order of the next product's k slots (see file comment).
template <typename T> struct FragFromAcc;
template <> struct FragFromAcc<bf16> {
  __device__ __forceinline__ static bf16x8 get(const f32x16& v, int t) {
    bf16x8 f;
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = (bf16)v[8 * t + i];
    return f;
  }
};
template <> struct FragFromAcc<float> {
  __device__ __forceinline__ static float get(const f32x16& v, int t) { return v[t]; }
};

// ----------------------------------------------------- global -> regs --
// B-operand fragments of one matrix row (row index = accumulator column c):
// for k-step t the lane holds columns [t*2KP + h*KP, +KP). `flip` XORs the
// sign bits (used to negate Q when the scale is negative). Rows >= n read 0.
template <typename T, int D> struct RowFrags;
template <int D> struct RowFrags<bf16, D> {
  static constexpr int TD = D / 16;
  bf16x8 f[TD];
  __device__ __forceinline__ void load(const bf16* g, int row, int n, int h, uint32_t flip) {
#pragma unroll
    for (int t = 0; t < TD; ++t) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (row < n) x = *(const u32x4*)(g + (size_t)row * D + 16 * t + 8 * h);
      x ^= (u32x4){flip, flip, flip, flip};
      f[t] = __builtin_bit_cast(bf16x8, x);
    }
  }
};
template <int D> struct RowFrags<float, D> {
  static constexpr int TD = D / 2;
  float f[TD];
  __device__ __forceinline__ void load(const float* g, int row, int n, int h, uint32_t flip) {
#pragma unroll
    for (int t = 0; t < TD; ++t) {
      uint32_t x = 0u;
      if (row < n) x = __float_as_uint(g[(size_t)row * D + 2 * t + h]);
      f[t] = __uint_as_float(x ^ flip);
    }
  }
};

// ---------------------------------------------------------- LDS tiles --
// Padded form of the 32-wide bf16 tiles at d = 128 (P = true below): stored
// rows of 20 16-byte chunk positions (16 data chunks, 4 spare), data chunk j
// of stored row s at position j ^ key32(s). The bank slot of a chunk is
// (20 s + (j ^ key32(s))) mod 16 = (4 s + (j ^ key32(s))) mod 16: the row
// read's 16 lanes of a pass fall into 4 classes of s mod 4 (distinct
// multiples of 4) and key32 separates the 4 rows of a class; the transposed
// read's 4 consecutive rows share one key and land on distinct multiples of
// 4. Both stay conflict-free, as with swz, but the swizzle only touches the
// two low chunk bits, so a lane's address for k step t or column block db is
// one of two bases plus an immediate offset instead of one register per t
// or db. The cost is 25 % more LDS (80 KB for the two K/V stages).
template <int D> struct Pad32 {
  static_assert(D == 128, "the padded 32-wide layout is laid out for d = 128");
  static constexpr int S = D / 8 + 4;   // chunk positions per stored row
  static constexpr int LD = 8 * S;      // row stride (elements)
};
__host__ __device__ constexpr int key32(int s) { return (s >> 2) & 3; }

// A ROWS x D tile, row stride LD = D + PAD elements (P: Pad32<D>::LD), rows
// permuted by srow.
template <typename T, int ROWS, int D, bool P = false> struct Tile {
  using E = Elem<T>;
  static_assert(!P || (sizeof(T) == 2 && D == 128), "the padded 32-wide layout is for bf16 at d = 128");
  static constexpr int LD = P ? 8 * (D / 8 + 4) : D + E::PAD;   // P: Pad32<D>::LD
  static constexpr int ELEMS = ROWS * LD;
  static constexpr int CPR = D / E::CH;            // 16-byte chunks per row
  static constexpr int NCH = ROWS * CPR;
  static constexpr int NPT = (NCH + 255) / 256;    // chunks per thread
};

// Register staging of one tile: global -> registers (issued early) and
// registers -> LDS (after the current tile's reads are done). Rows >= n read
// as zeros. Used for float32 tiles (padded rows).
template <typename T, int ROWS, int D> struct Stage {
  using TL = Tile<T, ROWS, D>;
  u32x4 r[TL::NPT];
  __device__ __forceinline__ void load(const T* g, int row0, int n, int tid) {
#pragma unroll
    for (int i = 0; i < TL::NPT; ++i) {
      const int ci = tid + 256 * i;
      u32x4 x = {0u, 0u, 0u, 0u};
      if (TL::NCH % 256 == 0 || ci < TL::NCH) {
        const int row = ci / TL::CPR, cc = ci % TL::CPR;
        if (row0 + row < n) x = *(const u32x4*)(g + (size_t)(row0 + row) * D + cc * Elem<T>::CH);
      }
      r[i] = x;
    }
  }
  __device__ __forceinline__ void store(T* s, int tid) const {
#pragma unroll
    for (int i = 0; i < TL::NPT; ++i) {
      const int ci = tid + 256 * i;
      if (TL::NCH % 256 == 0 || ci < TL::NCH) {
        const int row = ci / TL::CPR, cc = ci % TL::CPR;
        T* p = s + srow(row) * TL::LD + cc * Elem<T>::CH;
#pragma unroll
        for (int e = 0; e < 4; ++e) ((uint32_t*)p)[e] = r[i][e];
      }
    }
  }
};

// LDS DMA through the buffer path (buffer_load_dword / _dwordx4 ... lds):
// each lane's `size` bytes at byte offset `off` from the wave-uniform `base`
// land at lane * size from `lds`. The copies use the buffer form rather than
// global_load_lds because the latter is a FLAT instruction: while a FLAT
// copy into LDS is in flight the compiler cannot count LDS reads separately
// and waits for all of them (lgkmcnt(0)) before the first use, so every
// operand read of a step that overlaps the next tile's copy would expose its
// full latency. Offsets stay far below the 2^31-byte range of the resource.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t dma_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, unsigned off, ATTN_LDS void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, off, 0, 0, 0);
}
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t r, unsigned off, ATTN_LDS void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 4, off, 0, 0, 0);
}

// Global -> LDS transfer of one ROWS x D tile by a 4-wave workgroup.
// issue() starts the copy of rows [row0, row0 + ROWS) into `lds`; commit()
// finishes it (the caller's __syncthreads makes it visible).
//  * bf16: a 16-byte LDS DMA per lane (dma16), which writes each lane's 16 bytes at
//    lane * 16 of a 1 KB wave-contiguous LDS block; every lane fetches the
//    global chunk that belongs at its LDS slot (row permutation srow and
//    chunk swizzle swz applied on the global side), so no registers and no
//    LDS write instructions are spent. Rows >= n fetch row n - 1 instead
//    (finite values; the kernels mask those rows).
//  * float32: register staging (Stage), rows >= n as zeros.
template <typename T, int ROWS, int D, bool P = false> struct TileLoader;
template <int ROWS, int D> struct TileLoader<bf16, ROWS, D> {
  static constexpr int C = D / 8;                        // 16-byte chunks per row
  static constexpr int NI = ROWS * D * 2 / (4 * 1024);   // wave instructions per tile
  static_assert(NI >= 1 && ROWS * D * 2 == NI * 4096, "tile must split into 1 KB wave blocks");
  int off[NI];   // element offset of this lane's chunk inside the tile
  int xr[NI];    // its logical row
  __device__ __forceinline__ TileLoader(int w, int lane) {
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int L = 64 * (w * NI + j) + lane;
      const int s = L / C, slot = L % C;
      const int q = slot ^ swz<D>(s);
      const int x = (s & ~31) | perm32(s & 31);
      xr[j] = x;
      off[j] = x * D + 8 * q;
    }
  }
  __device__ __forceinline__ void issue(bf16* lds, const bf16* g, int row0, int n, int w) const {
    const bool full = row0 + ROWS <= n;
    const auto rs = dma_rsrc(g + (size_t)row0 * D);
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      int o = off[j];
      if (!full && row0 + xr[j] >= n) o -= (row0 + xr[j] - (n - 1)) * D;
      dma16(rs, 2u * (unsigned)o, (ATTN_LDS void*)(lds + 512 * (w * NI + j)));
    }
  }
  __device__ __forceinline__ void commit(bf16*) const {}
};
// bf16, padded layout: 1 KB wave copies over the tile's chunk positions
// (wave w issues copies w*NI + [0, NI)); lanes on a spare chunk take a byte
// offset beyond the buffer's range, which the buffer unit drops without a
// memory access. Rows >= n fetch row n - 1.
template <int ROWS, int D> struct TileLoader<bf16, ROWS, D, true> {
  static constexpr int C = D / 8, S = Pad32<D>::S;
  static constexpr int TI = ROWS * S / 64;          // wave copies per tile
  static constexpr int NI = TI / 4;                 // per wave (4-wave workgroups)
  static constexpr unsigned kSpare = 0x80000000u;   // out-of-range byte offset
  static_assert(NI * 4 * 64 == ROWS * S, "tile must split evenly into 1 KB wave copies");
  unsigned off[NI];   // byte offset of the lane's chunk in the global rows, kSpare on a spare chunk
  int xr[NI];         // its logical row
  __device__ __forceinline__ TileLoader(int w, int lane) {
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int L = 64 * (w * NI + j) + lane;   // chunk position in the tile
      const int s = L / S, pos = L % S;
      const int x = (s & ~31) | perm32(s & 31);
      xr[j] = x;
      off[j] = pos < C ? 2u * (unsigned)(x * D + 8 * (pos ^ key32(s))) : kSpare;
    }
  }
  __device__ __forceinline__ void issue(bf16* lds, const bf16* g, int row0, int n, int w) const {
    const auto rs = dma_rsrc(g + (size_t)row0 * D);
    if (row0 + ROWS <= n) {
#pragma unroll
      for (int j = 0; j < NI; ++j) dma16(rs, off[j], (ATTN_LDS void*)(lds + 512 * (w * NI + j)));
    } else {
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        unsigned o = off[j];
        const int over = row0 + xr[j] - (n - 1);
        if (o != kSpare && over > 0) o -= 2u * (unsigned)(over * D);
        dma16(rs, o, (ATTN_LDS void*)(lds + 512 * (w * NI + j)));
      }
    }
  }
  __device__ __forceinline__ void commit(bf16*) const {}
};
template <int ROWS, int D> struct TileLoader<float, ROWS, D> {
  Stage<float, ROWS, D> st;
  int tid;
  __device__ __forceinline__ TileLoader(int w, int lane) : tid(64 * w + lane) {}
  __device__ __forceinline__ void issue(float*, const float* g, int row0, int n, int) {
    st.load(g, row0, n, tid);
  }
  __device__ __forceinline__ void commit(float* lds) const { st.store(lds, tid); }
};

// Row read: A operand = logical rows of 32-row block `rb` (stored row
// 32*rb + c), k-step t over d.
template <typename T, int D, bool P = false> struct RowRead;
template <int D> struct RowRead<bf16, D> {
  __device__ __forceinline__ static bf16x8 get(const bf16* s, int rb, int t, int h, int c) {
    return *(const bf16x8*)(s + (32 * rb + c) * D + (((2 * t + h) ^ swz<D>(c)) * 8));
  }
};
// Padded layout: data chunk 2t + h sits at 4 (t >> 1) + ((2 (t & 1) + h) ^
// key32(c)), so the lane needs one base per parity of t. The lane part is
// clamped to its largest value (a no-op), as in TransRead.
template <int D> struct RowRead<bf16, D, true> {
  static constexpr int LD = Pad32<D>::LD;
  __device__ __forceinline__ static bf16x8 get(const bf16* s, int rb, int t, int h, int c) {
    const int lp = min(c * LD + 8 * ((2 * (t & 1) + h) ^ key32(c)), 31 * LD + 24);
    return *(const bf16x8*)(s + 32 * rb * LD + 16 * (t & ~1) + lp);
  }
};
template <int D> struct RowRead<float, D> {
  static constexpr int LD = D + Elem<float>::PAD;
  __device__ __forceinline__ static float get(const float* s, int rb, int t, int h, int c) {
    return s[(32 * rb + c) * LD + 2 * t + h];
  }
};

// Transposed read: A operand = column 32*db + c of the tile, contraction over
// logical rows of block rb; k-step t covers logical rows 16h + t*KP + [0, KP).
// The bf16 tiles hold ROWS rows. swz depends only on the low 4 bits of the
// stored row, which 32*rb + 16*t leave alone, so the lane's offset inside a
// 16-row group (swizzle included) depends on db and the lane only; rb and t
// add a constant, which becomes the read's immediate offset. The lane part is
// clamped to its largest value (a no-op): with the bound visible, the compiler
// can tell these reads from the LDS DMA into the other stage and does not wait
// for it.
template <typename T, int D, int ROWS = 64, bool P = false> struct TransRead;
template <int D, int ROWS> struct TransRead<bf16, D, ROWS> {
  // offset of lane (h, c) for column block db in the 16 stored rows starting
  // at a multiple of 16; hi selects the upper 4 logical rows (stored +8)
  __device__ __forceinline__ static int lane_off(int db, int h, int c, int hi) {
    // 16-lane group: source lane q = c % 16 reads stored row base + q/4 and
    // columns [32db + 16*(c/16) + 4*(q%4), +4); the transpose hands lane c
    // column 32db + c of those 4 rows.
    const int q = c & 15;
    const int r = 4 * h + (q >> 2) + 8 * hi;                // logical 16h+8t+k -> stored 16t+4h+k
    const int ch = 4 * db + 2 * (c >> 4) + ((q & 3) >> 1);  // 16-byte chunk of the columns
    return min(r * D + ((ch ^ swz<D>(r)) * 8) + (q & 1) * 4, 16 * D - 4);
  }
  __device__ __forceinline__ static bf16x8 get(const bf16* s, int rb, int db, int t, int h, int c) {
    const bf16* b = s + (32 * rb + 16 * t) * D;
    i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(b + lane_off(db, h, c, 0)));
    i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(b + lane_off(db, h, c, 1)));
    // whole-register bit casts (element-wise 16-bit inserts are avoided)
    const u32x2 a = __builtin_bit_cast(u32x2, lo), e = __builtin_bit_cast(u32x2, hi);
    return __builtin_bit_cast(bf16x8, (u32x4){a[0], a[1], e[0], e[1]});
  }
};
// Padded layout: the 4 rows a lane group reads share one key32, which only
// permutes the chunks inside an aligned group of 4, so column block db is an
// immediate offset (32 db) and the lane needs one base per half (rows +0 and
// +8 of the 16-row group).
template <int D, int ROWS> struct TransRead<bf16, D, ROWS, true> {
  static constexpr int LD = Pad32<D>::LD;
  __device__ __forceinline__ static int lane_off(int h, int c, int hi) {
    const int q = c & 15;
    const int r = 4 * h + (q >> 2) + 8 * hi;                // stored row in the 16-row group
    const int jj = 2 * (c >> 4) + ((q & 3) >> 1);           // chunk inside the aligned group of 4
    return min(r * LD + 8 * (jj ^ key32(r)) + (q & 1) * 4, 15 * LD + 28);
  }
  __device__ __forceinline__ static bf16x8 get(const bf16* s, int rb, int db, int t, int h, int c) {
    const bf16* b = s + (32 * rb + 16 * t) * LD + 32 * db;
    i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(b + lane_off(h, c, 0)));
    i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(b + lane_off(h, c, 1)));
    const u32x2 a = __builtin_bit_cast(u32x2, lo), e = __builtin_bit_cast(u32x2, hi);
    return __builtin_bit_cast(bf16x8, (u32x4){a[0], a[1], e[0], e[1]});
  }
};
template <int D, int ROWS> struct TransRead<float, D, ROWS> {
  static constexpr int LD = D + Elem<float>::PAD;
  __device__ __forceinline__ static float get(const float* s, int rb, int db, int t, int h, int c) {
    return s[(32 * rb + perm32_inv(16 * h + t)) * LD + 32 * db + c];
  }
};

// ------------------------------------------------- 16x16x32 variant --
// v_mfma_f32_16x16x32_bf16 (lane l, group g = l / 16, c = l % 16):
//   A: row c, k slots 8g + [0, 8); B: col c, same slots; accumulator: col c,
//   rows 4g + [0, 4).
// Chaining two 16-row accumulator blocks (rows 4g + j and 16 + 4g + j) into
// one operand gives every lane group the k slots of 8 rows that come as two
// runs of 4 consecutive rows, which is exactly what two ds_read_b64_tr_b16
// return. Tiles for this variant keep rows in natural order; their 16-byte
// chunks are swizzled with swz16 so that 16 consecutive rows of one chunk
// (row reads) and 8 consecutive rows of two adjacent chunks (transposed
// reads, per half-wave) each land on distinct bank slots.
__device__ __forceinline__ void mma16(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}

// On gfx950 a ds_read_b64 (also _tr_b16) serves each half-wave in one pass;
// a ds_read_b128 serves the 16 lanes that share bit 5 and the parity of
// bits 2, 3, 4 of the lane index (measured with single lane pairs), so the
// row read of this variant puts lanes (g, c) with g0 = parity(c2, c3) + const
// together; these swizzles are conflict-free for both patterns.
template <int D> __host__ __device__ constexpr int swz16(int s) {
  return D == 128 ? 2 * (s & 7)
       : D == 64  ? 2 * ((s >> 1) & 3)
                  : 2 * ((s >> 2) & 1);
}

// Global -> LDS DMA of a ROWS x D bf16 tile (natural row order, swz16
// chunks) by NW waves: 1 KB wave instructions, instruction i issued by wave
// i % NW. Rows >= n fetch row n - 1.
template <int ROWS, int D, int NW> struct TileLoader16 {
  static constexpr int C = D / 8;
  static constexpr int TI = ROWS * D * 2 / 1024;          // wave instructions per tile
  static constexpr int NI = (TI + NW - 1) / NW;            // per wave (upper bound)
  static_assert(ROWS * D * 2 == TI * 1024, "tile must split into 1 KB wave blocks");
  int off[NI];
  int xr[NI];
  __device__ __forceinline__ TileLoader16(int w, int lane) {
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int L = 64 * (w + NW * j) + lane;   // 16-byte chunk slot in the tile
      const int s = L / C, slot = L % C;
      xr[j] = s;
      off[j] = s * D + 8 * (slot ^ swz16<D>(s));
    }
  }
  __device__ __forceinline__ void issue(bf16* lds, const bf16* g, int row0, int n, int w) const {
    const bool full = row0 + ROWS <= n;
    const auto rs = dma_rsrc(g + (size_t)row0 * D);
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      if (TI % NW == 0 || w + NW * j < TI) {
        int o = off[j];
        if (!full && row0 + xr[j] >= n) o -= (row0 + xr[j] - (n - 1)) * D;
        dma16(rs, 2u * (unsigned)o, (ATTN_LDS void*)(lds + 512 * (w + NW * j)));
      }
    }
  }
};

// Global -> LDS DMA of a ROWS x COLS block of a bf16 matrix with a runtime
// row stride `ld` (elements): the same LDS layout as TileLoader16<ROWS, COLS,
// NW> (natural rows, swz16<COLS> chunks), so tr_read16<COLS> reads it. `g`
// points at the block's first column in matrix row 0; rows >= n fetch row
// n - 1.
template <int ROWS, int COLS, int NW> struct BlockLoader16 {
  static constexpr int C = COLS / 8;
  static constexpr int TI = ROWS * COLS * 2 / 1024;
  static constexpr int NI = (TI + NW - 1) / NW;
  static_assert(ROWS * COLS * 2 == TI * 1024, "block must split into 1 KB wave blocks");
  int off[NI];
  int xr[NI];
  int ld;
  __device__ __forceinline__ BlockLoader16(int w, int lane, int ld_) : ld(ld_) {
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int L = 64 * (w + NW * j) + lane;
      const int s = L / C, slot = L % C;
      xr[j] = s;
      off[j] = s * ld + 8 * (slot ^ swz16<COLS>(s));
    }
  }
  __device__ __forceinline__ void issue(bf16* lds, const bf16* g, int row0, int n, int w) const {
    const bool full = row0 + ROWS <= n;
    const auto rs = dma_rsrc(g + (size_t)row0 * ld);
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      if (TI % NW == 0 || w + NW * j < TI) {
        int o = off[j];
        if (!full && row0 + xr[j] >= n) o -= (row0 + xr[j] - (n - 1)) * ld;
        dma16(rs, 2u * (unsigned)o, (ATTN_LDS void*)(lds + 512 * (w + NW * j)));
      }
    }
  }
};

// Row read (16-wide): A operand = tile rows 16*rb + c, k-step t covers
// d in [32t, 32t + 32), lane group g takes d in [32t + 8g, +8).
template <int D>
__device__ __forceinline__ bf16x8 row_read16(const bf16* s, int rb, int t, int g, int c) {
  const int r = 16 * rb + c;
  return *(const bf16x8*)(s + r * D + 8 * ((4 * t + g) ^ swz16<D>(r)));
}

// Transposed read (16-wide): A operand = columns 16*db + c, k slots = rows
// r0 + 4g + [0, 4) and r0 + 16 + 4g + [0, 4) of a ROWS x D tile. Each whole
// offset is masked with the tile size minus one (a no-op on valid indexes,
// the tile size being a power of two), so the compiler sees every read stay
// inside the tile; TransRead and the padded reads instead clamp only the
// lane's part of the offset.
template <int D, int ROWS>
__device__ __forceinline__ bf16x8 tr_read16(const bf16* s, int r0, int db, int g, int c) {
  static_assert((ROWS * D & (ROWS * D - 1)) == 0, "tile size must be a power of two");
  constexpr int MASK = ROWS * D - 1;
  const int ra = r0 + 4 * g + (c >> 2);
  const int rb2 = ra + 16;
  const int ch = 2 * db + ((c & 3) >> 1);
  const int sub = (c & 1) * 4;
  const bf16* p0 = s + ((ra * D + 8 * (ch ^ swz16<D>(ra)) + sub) & MASK);
  const bf16* p1 = s + ((rb2 * D + 8 * (ch ^ swz16<D>(rb2)) + sub) & MASK);
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(p0));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(p1));
  const u32x2 x = __builtin_bit_cast(u32x2, lo), y = __builtin_bit_cast(u32x2, hi);
  return __builtin_bit_cast(bf16x8, (u32x4){x[0], x[1], y[0], y[1]});
}

// Padded 16-wide tiles: rows in natural order, chunks in natural order, row
// stride D + 16 elements (two spare 16-byte chunks). Chunk j of row r sits at
// bank slot (r (D/8 + 2) + j) mod 16, and (D/8 + 2)/2 is odd for D = 32, 64,
// 128, so 8 consecutive rows start on 8 distinct even slots: the row read (16
// rows of one chunk; rows r and r + 8 fall in one pass only with lanes of
// different parity, which take adjacent chunks) and the transposed read (8
// rows x 2 adjacent chunks per half-wave) are conflict-free, as with swz16.
// Unlike the swizzle, a lane's address for k step t or column block db is its
// own base plus a constant, so the reads of a tile share one address register
// and differ only in their immediate offsets.
template <int D> struct Pad16 {
  static constexpr int RS = D + 16;          // row stride (elements)
  static constexpr int C = D / 8, CP = C + 2; // data chunks and chunk positions per row
};

// Global -> LDS DMA of a ROWS x D bf16 tile into the padded layout by NW
// waves: 1 KB wave instructions over the tile's chunk positions, instruction
// i issued by wave i % NW. Lanes on a spare chunk take a byte offset beyond
// the buffer's range, which the buffer unit drops without a memory access
// (no branch, so the copies stay in the scheduling region of the loop
// body). Rows >= n fetch row n - 1.
template <int ROWS, int D, int NW> struct TileLoader16P {
  static constexpr int CP = Pad16<D>::CP, C = Pad16<D>::C;
  static constexpr int TI = ROWS * CP / 64;                // wave instructions per tile
  static constexpr int NI = (TI + NW - 1) / NW;            // per wave (upper bound)
  static constexpr unsigned kSpare = 0x80000000u;          // out-of-range byte offset
  static constexpr unsigned kRowBytes = 2u * D;
  static_assert(ROWS * CP == TI * 64, "tile must split into 1 KB wave blocks");
  static_assert((D & (D - 1)) == 0, "D must be a power of two");
  unsigned off[NI];   // byte offset of the lane's chunk in the global rows, kSpare on a spare chunk
  __device__ __forceinline__ TileLoader16P(int w, int lane) {
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int P = 64 * (w + NW * j) + lane;   // chunk position in the tile
      const int s = P / CP, slot = P % CP;
      off[j] = slot < C ? kRowBytes * s + 16u * slot : kSpare;
    }
  }
  __device__ __forceinline__ void issue(bf16* lds, const bf16* g, int row0, int n, int w) const {
    const auto rs = dma_rsrc(g + (size_t)row0 * D);
    if (row0 + ROWS <= n) {
#pragma unroll
      for (int j = 0; j < NI; ++j)
        if (TI % NW == 0 || w + NW * j < TI) dma16(rs, off[j], (ATTN_LDS void*)(lds + 512 * (w + NW * j)));
    } else {
      const int last = n - 1 - row0;   // last valid row of the tile
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        if (TI % NW == 0 || w + NW * j < TI) {
          unsigned o = off[j];
          const int over = (int)(o / kRowBytes) - last;
          if (o < kSpare && over > 0) o -= (unsigned)over * kRowBytes;
          dma16(rs, o, (ATTN_LDS void*)(lds + 512 * (w + NW * j)));
        }
      }
    }
  }
};

// Row read of a padded tile: A operand = rows 16*rb + c, k-step t covers d in
// [32t, 32t + 32), lane group g takes d in [32t + 8g, +8). The lane's part of
// the offset is clamped to its largest value (a no-op) so that alias analysis
// sees every read stay inside the tile; without that bound the compiler
// cannot tell the reads from DMA copies in flight into the other stage and
// waits for those copies first. The rest of the offset is an immediate.
template <int D>
__device__ __forceinline__ bf16x8 row_read16p(const bf16* s, int rb, int t, int g, int c) {
  constexpr int RS = Pad16<D>::RS;
  const int lp = min(c * RS + 8 * g, 15 * RS + 24);
  return *(const bf16x8*)(s + lp + 16 * rb * RS + 32 * t);
}

// Transposed read of a padded tile: A operand = columns 16*db + c, k slots =
// rows r0 + 4g + [0, 4) and r0 + 16 + 4g + [0, 4); lane (g, c) reads 4
// elements at column 16*db + 4*(c & 3) of rows r0 + 4g + (c >> 2) and 16
// rows further (lane part clamped as in row_read16p).
template <int D>
__device__ __forceinline__ bf16x8 tr_read16p(const bf16* s, int r0, int db, int g, int c) {
  constexpr int RS = Pad16<D>::RS;
  const int lp = min((4 * g + (c >> 2)) * RS + 4 * (c & 3), 15 * RS + 12);
  const bf16* p0 = s + lp + r0 * RS + 16 * db;
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(p0));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS i16x4*)(p0 + 16 * RS));
  const u32x2 x = __builtin_bit_cast(u32x2, lo), y = __builtin_bit_cast(u32x2, hi);
  return __builtin_bit_cast(bf16x8, (u32x4){x[0], x[1], y[0], y[1]});
}

// bf16 operand from two 16-row accumulator blocks (slots 0-3 from `a`,
// 4-7 from `b`).
__device__ __forceinline__ bf16x8 frag16(const f32x4& a, const f32x4& b) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = (bf16)a[i];
    f[4 + i] = (bf16)b[i];
  }
  return f;
}

// ------------------------------------------------------ output stores --
// Accumulator of a transposed product: lane (h, c) holds, for j-quad a,
// 4 consecutive columns 32*db + 8a + 4h + [0, 4) of its row.
template <typename T> struct Quad;
template <> struct Quad<bf16> {
  __device__ __forceinline__ static void store(bf16* p, float a, float b, float c, float d) {
    *(u32x2*)p = (u32x2){pack_bf16x2(a, b), pack_bf16x2(c, d)};
  }
  __device__ __forceinline__ static f32x4 load(const bf16* p) {
    const u32x2 x = *(const u32x2*)p;
    return (f32x4){__uint_as_float(x[0] << 16), __uint_as_float(x[0] & 0xffff0000u),
                   __uint_as_float(x[1] << 16), __uint_as_float(x[1] & 0xffff0000u)};
  }
};
template <> struct Quad<float> {
  __device__ __forceinline__ static void store(float* p, float a, float b, float c, float d) {
    *(f32x4*)p = (f32x4){a, b, c, d};
  }
  __device__ __forceinline__ static f32x4 load(const float* p) { return *(const f32x4*)p; }
};

// 16 consecutive row elements (an accumulator column j = 0..15 of one lane)
// rounded to T and packed as NC 16-byte chunks (element order = memory order).
template <typename T> struct Run16;
template <> struct Run16<bf16> {
  static constexpr int NC = 2;
  __device__ __forceinline__ static void pack(const f32x16& v, u32x4 (&r)[NC]) {
#pragma unroll
    for (int e = 0; e < NC; ++e)
      r[e] = (u32x4){pack_bf16x2(v[8 * e], v[8 * e + 1]), pack_bf16x2(v[8 * e + 2], v[8 * e + 3]),
                     pack_bf16x2(v[8 * e + 4], v[8 * e + 5]), pack_bf16x2(v[8 * e + 6], v[8 * e + 7])};
  }
};
template <> struct Run16<float> {
  static constexpr int NC = 4;
  __device__ __forceinline__ static void pack(const f32x16& v, u32x4 (&r)[NC]) {
#pragma unroll
    for (int e = 0; e < NC; ++e)
      r[e] = (u32x4){__float_as_uint(v[4 * e]), __float_as_uint(v[4 * e + 1]), __float_as_uint(v[4 * e + 2]),
                     __float_as_uint(v[4 * e + 3])};
  }
};
template <typename T>
__device__ __forceinline__ void store_run16(T* p, const u32x4 (&r)[Run16<T>::NC]) {
#pragma unroll
  for (int e = 0; e < Run16<T>::NC; ++e) *(u32x4*)(p + e * Elem<T>::CH) = r[e];
}

// --------------------------------------------------------- scheduling --
// Workgroup id -> (head, tile). Consecutive workgroup ids are dispatched
// round-robin over the 8 XCDs (each with its own L2); remapping gives every
// XCD a contiguous range of (head, tile) so the tiles of one head, which
// share K and V, run on the same L2. With `reverse`, tiles of a head are
// issued from the last (most work under a causal mask) to the first.
__device__ __forceinline__ void block_map(int bid, int nblocks, int ntiles, bool reverse,
                                          int& head, int& tile) {
  const int per = nblocks >> 3;
  int lin = bid;
  if (bid < per * 8) lin = (bid & 7) * per + (bid >> 3);
  head = lin / ntiles;
  const int t = lin - head * ntiles;
  tile = reverse ? ntiles - 1 - t : t;
}

}  // namespace attn
