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

constexpr int kWave = 64;
constexpr int kKeyTile = 64;      // keys per K/V tile of the row kernels (forward, dQ)
constexpr int kColKeys = 128;     // keys per workgroup of the column kernel (dK, dV)
constexpr int kQBlock = 32;       // query rows per step of the column kernel
constexpr int kLdsPad = 8;        // bf16 elements of padding per LDS row

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

}  // namespace kvs
