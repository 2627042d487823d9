// Device-side helpers shared by the gfx950 kernels of libkvs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
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

struct Trace {
  int tok0;  // first token of the trace in the packed layout
  int L;     // trace length
};

__device__ __forceinline__ Trace trace_of(const int* cu, int b, int T) {
  if (cu) {
    const int a = cu[b];
    return {a, cu[b + 1] - a};
  }
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

__device__ __forceinline__ float wave_xor32(float x) { return __shfl_xor(x, 32); }

// LDS tile of rows x D bf16 without padding.  Each row is D/8 chunks of 16
// bytes; chunk c of row r is stored at chunk position c ^ swz(r).  The
// permutation makes both access patterns of the MFMA operands free of bank
// conflicts: 16 lanes reading the same chunk of 16 consecutive rows (b128
// row reads), and 16-lane groups of the transposed read (4 rows x 32 bytes,
// two groups side by side).
template <int D>
struct Swz {
  static constexpr int CPR = D / 8;             // chunks per row
  static constexpr int RPL = kWave / CPR;       // rows covered by one 64-lane 16-byte-per-lane load
  __device__ static __forceinline__ int swz(int r) {
    return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
  }
  // element offset of (row r, column col) inside the tile
  __device__ static __forceinline__ int off(int r, int col) { return r * D + ((((col >> 3) ^ swz(r))) << 3) + (col & 7); }
};

// Issue asynchronous global -> LDS copies of tile rows [0, R) (global_load_lds_dwordx4:
// lane l of a wave writes 16 bytes at the wave's LDS base + 16 l).  Row r of the
// tile comes from global row min(row0 + r, rmax) (rows past the end of a trace
// repeat its last row; callers mask them).  Waves split the rows.
template <int D, int R>
__device__ __forceinline__ void stage_rows(uint16_t* lds, const uint16_t* __restrict__ g, long long row_stride,
                                           int row0, int rmax, int wave, int nwaves, int lane) {
  constexpr int RPL = Swz<D>::RPL;
  const int rl = lane / Swz<D>::CPR, p = lane % Swz<D>::CPR;
  for (int rb = wave * RPL; rb < R; rb += nwaves * RPL) {
    const int r = rb + rl;
    const int c = p ^ Swz<D>::swz(r);
    const int gr = min(row0 + r, rmax);
    const uint16_t* src = g + gr * row_stride + c * 8;
    __builtin_amdgcn_global_load_lds(src, (lds_void*)(lds + rb * D), 16, 0, 0);
  }
}

// 64 consecutive 4-byte values (clamped at index imax) into LDS, by one wave.
__device__ __forceinline__ void stage_words(void* lds, const void* __restrict__ g, int i0, int imax, int lane) {
  const int i = min(i0 + lane, imax);
  __builtin_amdgcn_global_load_lds((const char*)g + 4ll * i, (lds_void*)lds, 4, 0, 0);
}

// Wait for this wave's outstanding global loads (including LDS-direct ones).
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

}  // namespace kvs
