// Device-side helpers shared by the gfx950 kernels of libkvs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvs.h"

namespace kvs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) uint16_t lds_u16;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kWave = 64;
constexpr int kKeyTile = 64;      // keys per K/V tile of the row kernels (forward, dQ)
constexpr int kColKeys = 128;     // keys per workgroup of the column kernel (dK, dV)
constexpr int kQStep = 64;        // query rows staged per step of the column kernel

enum TileClass : int { kEmpty = 0, kPartial = 1, kFull = 2 };

// Class of the tile of rows [i0, i1) x keys [j0, j1) of one trace of length L,
// given the min and max of min(evict_at[j], L) over the tile's keys j < L.
// EMPTY : no (i, j) with i < L, j < L, j <= i < e_j.  Either every key lies
//         right of every row, or the tile is strictly below the diagonal and
//         no key survives to row i0.  (A tile that meets the diagonal always
//         holds the visible element (j, j), since e_j > j.)
// FULL  : all elements inside the trace, all left of or on the diagonal, and
//         every key still alive at the last row.
__device__ __forceinline__ int tile_class(int i0, int i1, int j0, int j1, int L, int emin, int emax) {
  const int i1c = min(i1, L), j1c = min(j1, L);
  if (j0 >= i1c) return kEmpty;
  if (j1c <= i0 && emax <= i0) return kEmpty;
  if (i1 <= L && j1 <= L && j1 <= i0 + 1 && emin >= i1) return kFull;
  return kPartial;
}

// Switches of the tile classifier, for internal-consistency checks: an EMPTY
// tile is processed (masked) instead of skipped; a FULL tile is masked
// element by element.  Either way every output must stay bit-identical.
constexpr int kFlagNoEmptySkip = KVS_FLAG_NO_EMPTY_SKIP;
constexpr int kFlagFullAsPartial = KVS_FLAG_FULL_AS_PARTIAL;

__host__ __device__ __forceinline__ int adjust_class(int c, int flags) {
  if ((flags & kFlagNoEmptySkip) && c == kEmpty) c = kPartial;
  if ((flags & kFlagFullAsPartial) && c == kFull) c = kPartial;
  return c;
}

struct Trace {
  int tok0;  // first token of the trace in the packed layout
  int L;     // trace length
};

// Trace b of a packed batch.  Offsets read from device memory are clamped, never
// trusted for addressing: tok0 to [0, ntok], the end to [tok0, ntok], and the
// length to T (max_seqlen, which sizes every grid), so a malformed cu_seqlens
// can give wrong results but no access outside the caller's buffers.
__host__ __device__ __forceinline__ Trace clamp_trace(int a, int z, int ntok, int T) {
  a = a < 0 ? 0 : (a > ntok ? ntok : a);
  z = z < a ? a : (z > ntok ? ntok : z);
  const int L = z - a;
  return {a, L < T ? L : T};
}

__device__ __forceinline__ Trace trace_of(const int* cu, int b, int T, int ntok) {
  if (cu) return clamp_trace(cu[b], cu[b + 1], ntok, T);
  return {b * T, T};
}

// Index of the per-key-tile statistics of tile kt of trace b (collision-free
// across traces: see the workspace layout in the host code).
__device__ __forceinline__ int kstat_index(int b, int tok0, int kt, int BN) { return b + tok0 / BN + kt; }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ bf16x8 lds_read_b128(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}

// LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane i supplies the address of 4 consecutive bf16; lane n receives element
// (n % 4) of the values read by lanes 4r + n / 4, r = 0..3.  When lane i of a
// group points at row (r0 + i / 4), column (c0 + 4 * (i % 4)) of a row-major
// tile, lane n receives column c0 + n of rows r0 .. r0 + 3.
__device__ __forceinline__ s16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)((lds_u16*)p));
}

__device__ __forceinline__ bf16x8 cat_tr(s16x4 lo, s16x4 hi) {
  s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// Eight fp32 accumulator values as one bf16 MFMA operand (round to nearest even).
__device__ __forceinline__ bf16x8 pack8(const f32x16& x, int base) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)x[base + e];
  return r;
}

__device__ __forceinline__ uint2 pack4_bf16(float a, float b, float c, float d) {
  bf16x4 r;
  r[0] = (__bf16)a;
  r[1] = (__bf16)b;
  r[2] = (__bf16)c;
  r[3] = (__bf16)d;
  return __builtin_bit_cast(uint2, r);
}

// Value of lane l ^ 32 (v_permlane32_swap: a VALU exchange of the two wave halves).
__device__ __forceinline__ float wave_xor32(float x) {
  // swap(x, x): first result = low half of x in both halves, second = high half in both
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}
// max and sum of x over lanes l and l ^ 32
__device__ __forceinline__ float halves_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Asynchronous global -> LDS copy (global_load_lds_dword{,x4}): lane l of the
// wave writes its 4 or 16 bytes at LDS byte address lds + (4 or 16) l.  Issued
// through inline assembly so that the compiler does not count the copy as an
// outstanding LDS access: with a compiler-visible LDS DMA in flight it waits for
// every earlier LDS read (lgkmcnt(0)) before each use of any of them.  Callers
// order the copies themselves (wait_vm() and a barrier before the tile is read).
// M0 holds the LDS base during the copy and is restored afterwards.
__device__ __forceinline__ uint32_t lds_addr(const void* lds) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void*)lds);
}
// base: wave-uniform global address; off: this lane's byte offset from it.
__device__ __forceinline__ void dma_b128(const void* base, uint32_t off, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"(lds)
      : "memory");
}
__device__ __forceinline__ void dma_b32(const void* base, uint32_t off, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"(lds)
      : "memory");
}
// Asynchronous copy of 16 bytes from this lane's own global address to LDS
// byte address lds + 16 l (gathers whose rows have no common base).
__device__ __forceinline__ void dma_b128_global(const void* src, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(lds)
      : "memory");
}
// Asynchronous copy of 4 bytes from this lane's own global address to LDS byte
// address lds + 4 l.
__device__ __forceinline__ void dma_b32_global(const void* src, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(lds)
      : "memory");
}
// A wave-uniform pointer held in scalar registers.
template <typename T>
__device__ __forceinline__ const T* uniform_ptr(const T* p) {
  const uint64_t u = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u), hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (const T*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// LDS tile of rows x D bf16 with padded rows and a per-row XOR on the
// 16-byte chunk index ("swizzle").  The hardware serves a b128 read 16 lanes
// at a time and a b64 read (the transposed operand reads) 32 lanes at a time,
// each group 256 bytes over the 64 four-byte banks, so two patterns must be
// conflict-free: 16 lanes reading one chunk of 16 consecutive rows (b128 MFMA
// operands) and 32 lanes reading a 4-row x 64-byte block (transposed reads).
//   wide (dK/dV tiles), D = 128: pitch 160 elements (20 chunks, 4 of them
//     padding), chunk ^= (r / 4) % 4.  Row r starts at bank 16 r (mod 64), so
//     4 consecutive rows cover all banks with 64 bytes each, and the XOR
//     spreads the 16 rows of a b128 group over 16 distinct 4-bank groups.
//   COMPACT (forward, dQ and decode tiles), D = 128: pitch 144, chunk ^=
//     (r / 8) % 2: b128 reads are conflict-free, transposed reads two-way
//     conflicted; 11% less LDS, which keeps two dQ workgroups on a CU and a
//     decode wave's double-buffered tiles within a quarter of the LDS.
//   D = 64: pitch 72, no swizzle.
// The swizzle touches only bits 0-1 of the chunk index and depends only on
// the row modulo 16, so moving by two k-steps (64 bytes), by 32-column blocks
// or by 16-row blocks is a constant offset: a b128 operand read is one of two
// per-lane bases (even or odd k-step) plus an immediate, a transposed read a
// per-lane base plus an immediate.
template <int D, bool COMPACT = false>
struct Lay {
  static constexpr int PITCH = D == 128 ? (COMPACT ? 144 : 160) : 72;   // bf16 elements per LDS row
  static constexpr int CPR = D / 8;                                   // 16-byte data chunks per row
  static constexpr int CPRP = PITCH / 8;                              // chunks per padded row
  __host__ __device__ static __forceinline__ int flip(int r) {
    return D == 128 ? (COMPACT ? ((r >> 3) & 1) : ((r >> 2) & 3)) : 0;
  }
  __host__ __device__ static __forceinline__ int off(int r, int col) { return r * PITCH + (((col >> 3) ^ flip(r)) << 3) + (col & 7); }
  // b128 operand reads: row (row0 + l % 32), columns 16 ks + 8 (l / 32) .. +7.
  // (odd k-steps: chunk bit 1 toggled, i.e. the base XOR 16, since rows
  // start at multiples of 32 elements)
  struct RowLane {
    int even;   // base of k-step 0 (row0 = 0)
  };
  __device__ static __forceinline__ RowLane row_lane(int lane) { return {off(lane & 31, 8 * (lane >> 5))}; }
  // element offset of k-step ks (add row0 * PITCH, row0 a multiple of 16)
  __device__ static __forceinline__ int row_at(RowLane rl, int ks) {
    const int odd = (D == 128 && !COMPACT) ? (rl.even ^ 16) : rl.even + 16;
    return (ks & 1 ? odd : rl.even) + 32 * (ks >> 1);
  }
  // transposed operand reads (see tr_operand): rows 4 (g16 / 2) + (li / 4) and +8,
  // columns 16 (g16 % 2) + 4 (li % 4); add row0 * PITCH + c0 (row0 % 16 == 0, c0 % 32 == 0).
  __device__ static __forceinline__ int tr_lo(int lane) {
    const int li = lane & 15, g16 = lane >> 4;
    return off(4 * (g16 >> 1) + (li >> 2), 16 * (g16 & 1) + 4 * (li & 3));
  }
  __device__ static __forceinline__ int tr_hi(int lane) {
    const int li = lane & 15, g16 = lane >> 4;
    return off(8 + 4 * (g16 >> 1) + (li >> 2), 16 * (g16 & 1) + 4 * (li & 3));
  }
};

// A operand of a 32x32x16 MFMA read transposed from an LDS tile: rows
// (contraction index) row0 + 4 half + {0..3} and row0 + 8 + 4 half + {0..3}
// (the order in which the C layout of a score block lists its 16 values),
// columns c0 + (l % 32).  tl, th = Lay<D, COMPACT>::tr_lo(lane), tr_hi(lane).
template <int D, bool COMPACT = false>
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* tile, int row0, int c0, int tl, int th) {
  const int o = row0 * Lay<D, COMPACT>::PITCH + c0;
  return cat_tr(lds_read_tr(tile + tl + o), lds_read_tr(tile + th + o));
}

// Asynchronous global -> LDS copies of an R-row tile (dma_b128:
// lane l of a wave writes 16 bytes at the wave's LDS base + 16 l, so the 64
// lanes of one instruction fill 64 consecutive 16-byte slots of the padded
// tile).  The NW waves of a workgroup take turns issuing the 64-slot pieces:
// wave w issues pieces w, w + NW, ...  The per-lane source offset of every
// piece is computed once (init).  Issuing a tile is one unsigned min and one
// copy per piece, with no branch but the wave's last piece when NW does not
// divide the piece count (a taken branch costs a wave tens of clocks, and the
// copies sit at the start of every tile step).  Rows past the end
// of a trace (row0 + r > rmax) all read the last 16 bytes of row rmax, a valid
// address; their values are never used unmasked (callers mask rows and keys
// past the trace end, and multiply them by exact zeros).  Lanes whose slot is
// row padding copy the row's first chunk into it (padding is never read).
template <int D, int R, int NW, bool COMPACT = false>
struct RowStager {
  using LY = Lay<D, COMPACT>;
  static constexpr int NI = R * LY::CPRP / kWave;   // 64-slot pieces per tile
  static constexpr int PW = (NI + NW - 1) / NW;      // pieces per wave (the last one conditional)
  static_assert(R * LY::CPRP % kWave == 0, "tile must fill whole 64-slot pieces");
  uint32_t off[PW];   // byte offset of the slot's source from the tile's first row (no clamping)

  // tile row and source element column of this lane's slot in piece n
  __host__ __device__ static __forceinline__ void slot(int n, int lane, int& r, int& col) {
    const int q = n * kWave + lane;
    r = q / LY::CPRP;
    const int pc = q - r * LY::CPRP;
    col = pc < LY::CPR ? 8 * (pc ^ LY::flip(r)) : 0;
  }
  // byte offset of the source of lane `lane`'s slot in piece n from the tile's first row (0 past the tile)
  __host__ __device__ static __forceinline__ uint32_t src_offset(int n, int lane, long long row_stride) {
    int r, col;
    slot(n, lane, r, col);
    return n < NI ? (uint32_t)(r * row_stride + col) * 2u : 0u;
  }
  // largest source offset of a tile whose last valid row is dr (= rmax - row0): the last 16 bytes of
  // that row; a slot of a row past dr has a larger offset (row_stride >= D), valid rows a smaller one
  __host__ __device__ static __forceinline__ uint32_t limit(int dr, long long row_stride) {
    return dr >= R - 1 ? 0xffffffffu : (uint32_t)(dr * row_stride + D - 8) * 2u;
  }
  // whether piece i of a wave (piece number n) exists
  __host__ __device__ static __forceinline__ bool issues(int i, int n) { return i < PW - 1 || NI % NW == 0 || n < NI; }

  __device__ __forceinline__ void init(int wave, int lane, long long row_stride) {
#pragma unroll
    for (int i = 0; i < PW; ++i) off[i] = src_offset(wave + i * NW, lane, row_stride);
  }
  // row0 <= rmax; rows row0 .. min(row0 + R - 1, rmax) of g span less than 4 GiB; row_stride as given to init().
  // lds: LDS byte address of the tile (lds_addr).
  __device__ __forceinline__ void issue(uint32_t lds, const uint16_t* __restrict__ g, long long row_stride, int row0,
                                        int rmax, int wave) const {
    const uint16_t* base = uniform_ptr(g + (long long)row0 * row_stride);
    const uint32_t lim = limit(rmax - row0, row_stride);
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int n = wave + i * NW;
      if (issues(i, n)) dma_b128(base, min(off[i], lim), lds + n * kWave * 16);
    }
  }
};

// 64 consecutive 4-byte values (clamped at index imax) into LDS, by one wave.
__device__ __forceinline__ void stage_words(uint32_t lds, const void* __restrict__ g, int i0, int imax, int lane) {
  const char* base = uniform_ptr((const char*)g + 4ll * i0);
  dma_b32(base, 4u * (uint32_t)(min(i0 + lane, imax) - i0), lds);
}

// Wait for this wave's outstanding global loads (including LDS-direct ones).
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

}  // namespace kvs
