// gfx950 kernels of libkvs: eviction-masked attention forward and backward.
//
// Mask (Section 2, "KV-streams"): query i of a trace sees key j iff
// j <= i < evict_at[j].  Kernels skip EMPTY tiles, run FULL tiles without
// mask arithmetic and mask PARTIAL tiles element by element.
//
// Row kernels (forward, dQ): a workgroup owns 32*TC query tokens of HG
// q-heads that share one KV head; each wave owns 32 tokens of one q-head.
// K/V tiles of 64 keys are staged once in LDS (double-buffered) and read by
// every wave of the workgroup, so the G heads of a GQA group share them.
// Scores are computed transposed, S^T = K Q^T (keys on the MFMA M axis,
// queries on N), so each lane holds 16 scores of a single query and the row
// max / row sum need one cross-lane exchange per tile.
//
// Column kernel (dK, dV): a workgroup owns 128 keys of one KV head (32 per
// wave, with K and V held in registers) and walks the contiguous range of
// query rows that can see any of them, for each q-head of the group; Q, dO,
// LSE and Delta blocks of 32 rows are staged in LDS.
//
// All MFMAs are v_mfma_f32_32x32x16_bf16 (bf16 in, fp32 accumulate).
// Operand layouts (per lane l, h = l / 32):  A[m = l%32][k = 8h .. 8h+7],
// B[k = 8h .. 8h+7][n = l%32], C[m = 8(r/4) + 4h + r%4][n = l%32], r = 0..15.
#include "kvs_device.h"
#include "kvs_launch.h"

#include <climits>

namespace kvs {

// ---------------------------------------------------------------- kernel arguments
struct RowArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int* evict;
  const int* cu;
  const int2* kstats;
  uint16_t* o;          // forward output
  float* lse;           // forward output
  const uint16_t* dout; // dQ kernel input
  const float* lse_in;  // dQ kernel input
  const float* delta;   // dQ kernel input
  uint16_t* dq;         // dQ kernel output
  int B, T, Hq, Hkv, G, HG, TC, nhg, nqt, ntok;
  int varlen;
  float scale_log2;     // softmax_scale * log2(e)
  float scale;
};

struct ColArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* dout;
  const float* lse;
  const float* delta;
  const int* evict;
  const int* cu;
  uint16_t* dk;
  uint16_t* dv;
  int B, T, Hq, Hkv, G, nkt, ntok;
  int varlen;
  float scale_log2;
  float scale;
};

// LSE / Delta layout: fixed [B][Hq][T], varlen [Hq][ntok].
__device__ __forceinline__ long long lse_index(int varlen, int ntok, int Hq, int T, int b, int h, int tok0, int i) {
  return varlen ? (long long)h * ntok + tok0 + i : ((long long)b * Hq + h) * T + i;
}

// ---------------------------------------------------------------- key-tile statistics
// min and max of min(evict_at[j], L) over the keys j < L of the tile [j0, j0 + BN).
__device__ __forceinline__ int2 key_tile_stats(const int* __restrict__ evict, const Trace& tr, int j0, int BN) {
  int mn = INT_MAX, mx = INT_MIN;
  const int j1 = min(j0 + BN, tr.L);
  for (int j = j0; j < j1; ++j) {
    const int e = min(evict[tr.tok0 + j], tr.L);
    mn = min(mn, e);
    mx = max(mx, e);
  }
  return make_int2(mn, mx);
}

// One thread per (trace, key tile of BN keys).
__global__ void __launch_bounds__(64) kstats_kernel(const int* __restrict__ evict, const int* __restrict__ cu,
                                                    int T, int BN, int2* __restrict__ out) {
  const int kt = blockIdx.x * kWave + threadIdx.x, b = blockIdx.y;
  const Trace tr = trace_of(cu, b, T);
  const int j0 = kt * BN;
  if (j0 >= tr.L) return;
  out[kstat_index(b, tr.tok0, kt, BN)] = key_tile_stats(evict, tr, j0, BN);
}

// ---------------------------------------------------------------- tile-class grid
// One thread per (trace, q-tile, k-tile); grids of all traces concatenated.
__global__ void __launch_bounds__(64) classify_kernel(const int* __restrict__ evict, const int* __restrict__ cu,
                                                      int B, int T, int BM, int BN, uint8_t* __restrict__ out) {
  const int kt = blockIdx.x * kWave + threadIdx.x;
  const int qt = blockIdx.y, b = blockIdx.z;
  const Trace tr = trace_of(cu, b, T);
  const int nq = (tr.L + BM - 1) / BM, nk = (tr.L + BN - 1) / BN;
  if (qt >= nq || kt >= nk) return;
  long long off = 0;
  for (int bb = 0; bb < b; ++bb) {
    const Trace t2 = trace_of(cu, bb, T);
    off += (long long)((t2.L + BM - 1) / BM) * ((t2.L + BN - 1) / BN);
  }
  const int2 st = key_tile_stats(evict, tr, kt * BN, BN);
  out[off + (long long)qt * nk + kt] =
      (uint8_t)tile_class(qt * BM, qt * BM + BM, kt * BN, kt * BN + BN, tr.L, st.x, st.y);
}

// ---------------------------------------------------------------- evict_at validation
__device__ unsigned long long g_first_bad;
__device__ int g_cu_bad;

__global__ void check_init_kernel() {
  g_first_bad = ULLONG_MAX;
  g_cu_bad = 0;
}

__global__ void __launch_bounds__(256) check_kernel(const int* __restrict__ evict, const int* __restrict__ cu,
                                                    int B, int T, int ntok) {
  const int b = blockIdx.y;
  if (cu) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      const int a = cu[b], z = cu[b + 1];
      if ((b == 0 && a != 0) || z < a || (b == B - 1 && z != ntok) || z > ntok) atomicOr(&g_cu_bad, 1);
    }
  }
  const Trace tr = trace_of(cu, b, T);
  if (tr.L <= 0 || tr.tok0 < 0 || tr.tok0 + tr.L > ntok) return;
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < tr.L; j += gridDim.x * blockDim.x) {
    if (evict[tr.tok0 + j] <= j) atomicMin(&g_first_bad, (unsigned long long)(tr.tok0 + j));
  }
}

// ---------------------------------------------------------------- key-tile walker
// Every wave of a workgroup walks the same sequence of non-EMPTY key tiles of
// its query rows [i0, i1): 64 candidate tiles are classified at a time (one
// per lane) and the results kept as two ballots.
struct TileWalker {
  int base, lim;
  unsigned long long live, full;
};

__device__ __forceinline__ void walker_load(TileWalker& w, const int2* __restrict__ ks, int kidx0, int i0, int i1,
                                            int L) {
  const int kt = w.base + (threadIdx.x & 63);
  bool ne = false, fu = false;
  if (kt < w.lim) {
    const int2 st = ks[kidx0 + kt];
    const int c = tile_class(i0, i1, kt * kKeyTile, kt * kKeyTile + kKeyTile, L, st.x, st.y);
    ne = c != kEmpty;
    fu = c == kFull;
  }
  w.live = __ballot(ne);
  w.full = __ballot(fu);
}

__device__ __forceinline__ int walker_next(TileWalker& w, const int2* __restrict__ ks, int kidx0, int i0, int i1,
                                           int L) {
  while (w.live == 0ull) {
    w.base += 64;
    if (w.base >= w.lim) return -1;
    walker_load(w, ks, kidx0, i0, i1, L);
  }
  const int bit = __builtin_ctzll(w.live);
  w.live &= w.live - 1ull;
  return w.base + bit;
}

// ---------------------------------------------------------------- K/V tile staging (row kernels)
template <int D>
struct KVStage {
  static constexpr int PITCH = D + kLdsPad;
  static constexpr int CPR = D / 8;                       // 16-byte chunks per row
  static constexpr int CHUNKS = kKeyTile * CPR;
  static constexpr int MAXC = (CHUNKS + 255) / 256;       // per thread, >= 4 waves per workgroup
  uint4 rk[MAXC], rv[MAXC];
  int re;

  __device__ __forceinline__ void load(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                                       const int* __restrict__ evict, const Trace& tr, int Hkv, int g, int kt,
                                       int tid, int nthr, bool with_v) {
    const int j0 = kt * kKeyTile;
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
      const int c = tid + u * nthr;
      if (c < CHUNKS) {
        const int r = c / CPR, cc = c % CPR;
        const int j = j0 + r;
        if (j < tr.L) {
          const size_t off = ((size_t)(tr.tok0 + j) * Hkv + g) * D + cc * 8;
          rk[u] = *reinterpret_cast<const uint4*>(K + off);
          if (with_v) rv[u] = *reinterpret_cast<const uint4*>(V + off);
        } else {
          rk[u] = make_uint4(0, 0, 0, 0);
          rv[u] = make_uint4(0, 0, 0, 0);
        }
      }
    }
    if (tid < kKeyTile) {
      const int j = j0 + tid;
      re = (j < tr.L) ? min(evict[tr.tok0 + j], tr.L) : 0;  // keys past the trace end are never visible
    }
  }

  __device__ __forceinline__ void store(uint16_t* sK, uint16_t* sV, int* sE, int tid, int nthr, bool with_v) {
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
      const int c = tid + u * nthr;
      if (c < CHUNKS) {
        const int r = c / CPR, cc = c % CPR;
        *reinterpret_cast<uint4*>(sK + r * PITCH + cc * 8) = rk[u];
        if (with_v) *reinterpret_cast<uint4*>(sV + r * PITCH + cc * 8) = rv[u];
      }
    }
    if (tid < kKeyTile) sE[tid] = re;
  }
};

// S^T block (32 keys x 32 queries) of the current tile: A = K rows from LDS, B = Q^T in registers.
template <int D>
__device__ __forceinline__ f32x16 scores_t(const uint16_t* sK, int kb, const bf16x8* qreg, int col, int half) {
  constexpr int PITCH = D + kLdsPad;
  f32x16 s = {};
  const uint16_t* base = sK + (32 * kb + col) * PITCH + 8 * half;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) s = mfma32(lds_read_b128(base + 16 * ks), qreg[ks], s);
  return s;
}

// Mask of a PARTIAL tile for S^T blocks: element r of block kb is key
// j = j0 + 32 kb + 8 (r/4) + 4 half + r%4 and query i.
__device__ __forceinline__ void mask_t(f32x16& s, const int* sE, int kb, int j0, int i, int L, int half) {
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4) {
    const int jl = 32 * kb + 8 * q4 + 4 * half;
    const int4 e4 = *reinterpret_cast<const int4*>(sE + jl);
    const int ev[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = j0 + jl + t;
      const bool vis = (j <= i) && (i < ev[t]) && (i < L);
      if (!vis) s[4 * q4 + t] = -INFINITY;
    }
  }
}

// A operand of a 32x32x16 MFMA read transposed from a row-major LDS tile:
// rows (contraction index) r0 + {0..3} and r0 + 8 + {0..3} with r0 = 16 t + 4 half
// (the order in which the C layout of a score block lists its 16 values),
// columns c0 + (l % 32).
template <int PITCH>
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* tile, int row0, int c0, int lane) {
  const int li = lane & 15, g16 = lane >> 4;
  const int r = row0 + 4 * (g16 >> 1) + (li >> 2);
  const int c = c0 + 16 * (g16 & 1) + 4 * (li & 3);
  const s16x4 lo = lds_read_tr(tile + r * PITCH + c);
  const s16x4 hi = lds_read_tr(tile + (r + 8) * PITCH + c);
  return cat_tr(lo, hi);
}

// Head grouping of a row-kernel workgroup.
struct RowTile {
  int g, h, b, i0, i1, i0w, hh;
  Trace tr;
};

__device__ __forceinline__ bool row_tile(const RowArgs& a, RowTile& t) {
  int wg = blockIdx.x;
  t.g = wg % a.Hkv;
  wg /= a.Hkv;
  const int hgrp = wg % a.nhg;
  wg /= a.nhg;
  t.b = wg % a.B;
  wg /= a.B;
  const int qt = a.nqt - 1 - wg;  // later query tiles see more keys: start them first
  t.tr = trace_of(a.cu, t.b, a.T);
  const int BMt = 32 * a.TC;
  t.i0 = qt * BMt;
  t.i1 = t.i0 + BMt;
  if (t.i0 >= t.tr.L) return false;
  const int wave = threadIdx.x >> 6;
  t.hh = wave % a.HG;
  t.h = t.g * a.G + hgrp * a.HG + t.hh;
  t.i0w = t.i0 + 32 * (wave / a.HG);
  return true;
}

// ---------------------------------------------------------------- forward
template <int D>
__global__ void __launch_bounds__(512) fwd_kernel(RowArgs a) {
  constexpr int KS = D / 16, DB = D / 32;
  using Stage = KVStage<D>;
  constexpr int PITCH = Stage::PITCH;
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kKeyTile * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][kKeyTile * PITCH];
  __shared__ __attribute__((aligned(16))) int sE[2][kKeyTile];

  RowTile rt;
  if (!row_tile(a, rt)) return;
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid & 63;
  const int half = lane >> 5, col = lane & 31;
  const Trace tr = rt.tr;
  const int i = rt.i0w + col;
  const bool row_ok = i < tr.L;

  bf16x8 qreg[KS];
  {
    const uint16_t* qrow = a.q + ((size_t)(tr.tok0 + (row_ok ? i : 0)) * a.Hq + rt.h) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = row_ok ? as_bf16x8(*reinterpret_cast<const uint4*>(qrow + 16 * ks)) : bf16x8{};
  }

  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) acc[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  const int kidx0 = kstat_index(rt.b, tr.tok0, 0, kKeyTile);
  TileWalker w{0, (min(rt.i1, tr.L) + kKeyTile - 1) / kKeyTile, 0ull, 0ull};
  walker_load(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L);
  int kt = walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L);

  Stage st;
  if (kt >= 0) {
    st.load(a.k, a.v, a.evict, tr, a.Hkv, rt.g, kt, tid, nthr, true);
    st.store(sK[0], sV[0], sE[0], tid, nthr, true);
  }
  __syncthreads();
  int buf = 0;
  while (kt >= 0) {
    const int nkt = walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L);
    if (nkt >= 0) st.load(a.k, a.v, a.evict, tr, a.Hkv, rt.g, nkt, tid, nthr, true);

    const int j0 = kt * kKeyTile;
    const int2 ks_ = a.kstats[kidx0 + kt];
    const int cls = tile_class(rt.i0w, rt.i0w + 32, j0, j0 + kKeyTile, tr.L, ks_.x, ks_.y);
    if (cls != kEmpty) {
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = scores_t<D>(sK[buf], kb, qreg, col, half);
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] *= a.scale_log2;
        if (cls == kPartial) mask_t(s[kb], sE[buf], kb, j0, i, tr.L, half);
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
      mx = fmaxf(mx, wave_xor32(mx));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(s[kb][r] - m_use);
          s[kb][r] = p;
          ls += p;
        }
      l_run = l_run * alpha + ls;
      m_run = m_new;
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[d][r] *= alpha;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8 pb = pack8(s[kb], 8 * t);
#pragma unroll
          for (int d = 0; d < DB; ++d)
            acc[d] = mfma32(tr_operand<PITCH>(sV[buf], 32 * kb + 16 * t, 32 * d, lane), pb, acc[d]);
        }
    }
    if (nkt >= 0) st.store(sK[buf ^ 1], sV[buf ^ 1], sE[buf ^ 1], tid, nthr, true);
    __syncthreads();
    buf ^= 1;
    kt = nkt;
  }

  const float l_tot = l_run + wave_xor32(l_run);
  if (row_ok) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    uint16_t* orow = a.o + ((size_t)(tr.tok0 + i) * a.Hq + rt.h) * D;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<uint2*>(orow + 32 * d + 8 * q4 + 4 * half) =
            pack4_bf16(acc[d][4 * q4] * inv, acc[d][4 * q4 + 1] * inv, acc[d][4 * q4 + 2] * inv,
                       acc[d][4 * q4 + 3] * inv);
    if (half == 0)
      a.lse[lse_index(a.varlen, a.ntok, a.Hq, a.T, rt.b, rt.h, tr.tok0, i)] =
          (m_run + __log2f(l_tot)) * 0.6931471805599453f;
  }
}

// ---------------------------------------------------------------- backward: Delta = rowsum(dO * O)
template <int D>
__global__ void __launch_bounds__(256) bwd_pre_kernel(const uint16_t* __restrict__ o, const uint16_t* __restrict__ dout,
                                                      float* __restrict__ delta, int ntok, int Hq, int T,
                                                      int varlen) {
  constexpr int PER = D / 16;  // elements per lane, 16 lanes per row
  const int sub = threadIdx.x & 15;
  const long long row = (long long)blockIdx.x * (blockDim.x / 16) + (threadIdx.x >> 4);
  const bool ok = row < (long long)ntok * Hq;
  float s = 0.f;
  if (ok) {
    const size_t off = (size_t)row * D + sub * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const float x = (float)__builtin_bit_cast(__bf16, o[off + e]);
      const float y = (float)__builtin_bit_cast(__bf16, dout[off + e]);
      s += x * y;
    }
  }
#pragma unroll
  for (int m = 8; m > 0; m >>= 1) s += __shfl_xor(s, m);
  if (ok && sub == 0) {
    const int tok = (int)(row / Hq), h = (int)(row % Hq);
    const long long idx = varlen ? (long long)h * ntok + tok : ((long long)(tok / T) * Hq + h) * T + tok % T;
    delta[idx] = s;
  }
}

// ---------------------------------------------------------------- backward: dQ (row kernel)
template <int D>
__global__ void __launch_bounds__(512) dq_kernel(RowArgs a) {
  constexpr int KS = D / 16, DB = D / 32;
  using Stage = KVStage<D>;
  constexpr int PITCH = Stage::PITCH;
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kKeyTile * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][kKeyTile * PITCH];
  __shared__ __attribute__((aligned(16))) int sE[2][kKeyTile];

  RowTile rt;
  if (!row_tile(a, rt)) return;
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid & 63;
  const int half = lane >> 5, col = lane & 31;
  const Trace tr = rt.tr;
  const int i = rt.i0w + col;
  const bool row_ok = i < tr.L;

  bf16x8 qreg[KS], oreg[KS];
  float lse2 = 0.f, dlt = 0.f;
  {
    const size_t roff = ((size_t)(tr.tok0 + (row_ok ? i : 0)) * a.Hq + rt.h) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qreg[ks] = row_ok ? as_bf16x8(*reinterpret_cast<const uint4*>(a.q + roff + 16 * ks)) : bf16x8{};
      oreg[ks] = row_ok ? as_bf16x8(*reinterpret_cast<const uint4*>(a.dout + roff + 16 * ks)) : bf16x8{};
    }
    if (row_ok) {
      const long long li = lse_index(a.varlen, a.ntok, a.Hq, a.T, rt.b, rt.h, tr.tok0, i);
      lse2 = a.lse_in[li] * 1.4426950408889634f;
      dlt = a.delta[li];
    }
  }

  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) acc[d] = f32x16{};

  const int kidx0 = kstat_index(rt.b, tr.tok0, 0, kKeyTile);
  TileWalker w{0, (min(rt.i1, tr.L) + kKeyTile - 1) / kKeyTile, 0ull, 0ull};
  walker_load(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L);
  int kt = walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L);

  Stage st;
  if (kt >= 0) {
    st.load(a.k, a.v, a.evict, tr, a.Hkv, rt.g, kt, tid, nthr, true);
    st.store(sK[0], sV[0], sE[0], tid, nthr, true);
  }
  __syncthreads();
  int buf = 0;
  while (kt >= 0) {
    const int nkt = walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L);
    if (nkt >= 0) st.load(a.k, a.v, a.evict, tr, a.Hkv, rt.g, nkt, tid, nthr, true);

    const int j0 = kt * kKeyTile;
    const int2 ks_ = a.kstats[kidx0 + kt];
    const int cls = tile_class(rt.i0w, rt.i0w + 32, j0, j0 + kKeyTile, tr.L, ks_.x, ks_.y);
    if (cls != kEmpty) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = scores_t<D>(sK[buf], kb, qreg, col, half);
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = s[r] * a.scale_log2 - lse2;
        if (cls == kPartial) mask_t(s, sE[buf], kb, j0, i, tr.L, half);
        f32x16 dp = scores_t<D>(sV[buf], kb, oreg, col, half);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(s[r]);
          s[r] = p * (dp[r] - dlt);
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8 dsb = pack8(s, 8 * t);
#pragma unroll
          for (int d = 0; d < DB; ++d)
            acc[d] = mfma32(tr_operand<PITCH>(sK[buf], 32 * kb + 16 * t, 32 * d, lane), dsb, acc[d]);
        }
      }
    }
    if (nkt >= 0) st.store(sK[buf ^ 1], sV[buf ^ 1], sE[buf ^ 1], tid, nthr, true);
    __syncthreads();
    buf ^= 1;
    kt = nkt;
  }

  if (row_ok) {
    uint16_t* drow = a.dq + ((size_t)(tr.tok0 + i) * a.Hq + rt.h) * D;
    const float sc = a.scale;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<uint2*>(drow + 32 * d + 8 * q4 + 4 * half) =
            pack4_bf16(acc[d][4 * q4] * sc, acc[d][4 * q4 + 1] * sc, acc[d][4 * q4 + 2] * sc,
                       acc[d][4 * q4 + 3] * sc);
  }
}

// ---------------------------------------------------------------- backward: dK, dV (column kernel)
template <int D>
__global__ void __launch_bounds__(256) dkdv_kernel(ColArgs a) {
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int PITCH = D + kLdsPad;
  constexpr int CPR = D / 8;
  constexpr int CHUNKS = kQBlock * CPR;       // per tensor
  constexpr int MAXC = (CHUNKS + 255) / 256;
  __shared__ __attribute__((aligned(16))) uint16_t sQ[2][kQBlock * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t sO[2][kQBlock * PITCH];
  __shared__ __attribute__((aligned(16))) float sL[2][kQBlock];
  __shared__ __attribute__((aligned(16))) float sD[2][kQBlock];
  __shared__ int sEmax[4];

  int wg = blockIdx.x;
  const int g = wg % a.Hkv;
  wg /= a.Hkv;
  const int b = wg % a.B;
  wg /= a.B;
  const int kt = wg;
  const Trace tr = trace_of(a.cu, b, a.T);
  const int j0 = kt * kColKeys;
  if (j0 >= tr.L) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;
  const int jw0 = j0 + 32 * wave;
  const int j = jw0 + col;
  const bool key_ok = j < tr.L;
  const int ej = key_ok ? min(a.evict[tr.tok0 + j], tr.L) : 0;
  int emin_w = key_ok ? ej : INT_MAX, emax_w = key_ok ? ej : INT_MIN;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    emin_w = min(emin_w, __shfl_xor(emin_w, off));
    emax_w = max(emax_w, __shfl_xor(emax_w, off));
  }
  if (lane == 0) sEmax[wave] = emax_w;

  bf16x8 kreg[KS], vreg[KS];
  {
    const size_t koff = ((size_t)(tr.tok0 + (key_ok ? j : 0)) * a.Hkv + g) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kreg[ks] = key_ok ? as_bf16x8(*reinterpret_cast<const uint4*>(a.k + koff + 16 * ks)) : bf16x8{};
      vreg[ks] = key_ok ? as_bf16x8(*reinterpret_cast<const uint4*>(a.v + koff + 16 * ks)) : bf16x8{};
    }
  }
  __syncthreads();
  const int emax_wg = max(max(sEmax[0], sEmax[1]), max(sEmax[2], sEmax[3]));
  const int qb_lo = j0 / kQBlock;
  const int qb_hi = (emax_wg + kQBlock - 1) / kQBlock;
  const int steps = (qb_hi - qb_lo) * a.G;

  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) {
    dk[d] = f32x16{};
    dv[d] = f32x16{};
  }

  uint4 rq[MAXC], ro[MAXC];
  float rl = 0.f;
  auto load = [&](int step) {
    const int qb = qb_lo + step / a.G;
    const int h = g * a.G + step % a.G;
    const int i0 = qb * kQBlock;
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
      const int c = tid + u * 256;
      if (c < CHUNKS) {
        const int r = c / CPR, cc = c % CPR;
        const int i = i0 + r;
        if (i < tr.L) {
          const size_t off = ((size_t)(tr.tok0 + i) * a.Hq + h) * D + cc * 8;
          rq[u] = *reinterpret_cast<const uint4*>(a.q + off);
          ro[u] = *reinterpret_cast<const uint4*>(a.dout + off);
        } else {
          rq[u] = make_uint4(0, 0, 0, 0);
          ro[u] = make_uint4(0, 0, 0, 0);
        }
      }
    }
    if (tid < 2 * kQBlock) {
      const int i = i0 + (tid & 31);
      if (i < tr.L) {
        const long long li = lse_index(a.varlen, a.ntok, a.Hq, a.T, b, h, tr.tok0, i);
        rl = (tid < kQBlock) ? a.lse[li] * 1.4426950408889634f : a.delta[li];
      } else {
        rl = 0.f;
      }
    }
  };
  auto store = [&](int bufi) {
#pragma unroll
    for (int u = 0; u < MAXC; ++u) {
      const int c = tid + u * 256;
      if (c < CHUNKS) {
        const int r = c / CPR, cc = c % CPR;
        *reinterpret_cast<uint4*>(&sQ[bufi][r * PITCH + cc * 8]) = rq[u];
        *reinterpret_cast<uint4*>(&sO[bufi][r * PITCH + cc * 8]) = ro[u];
      }
    }
    if (tid < kQBlock) sL[bufi][tid] = rl;
    else if (tid < 2 * kQBlock) sD[bufi][tid - kQBlock] = rl;
  };

  if (steps > 0) {
    load(0);
    store(0);
  }
  __syncthreads();
  int buf = 0;
  for (int step = 0; step < steps; ++step) {
    const bool more = step + 1 < steps;
    if (more) load(step + 1);
    const int qb = qb_lo + step / a.G;
    const int i0 = qb * kQBlock;
    const int cls = tile_class(i0, i0 + kQBlock, jw0, jw0 + 32, tr.L, emin_w, emax_w);
    if (cls != kEmpty) {
      // S = Q K^T (rows i, columns = this wave's 32 keys)
      f32x16 s = {};
      f32x16 dp = {};
      {
        const uint16_t* qb_ = &sQ[buf][col * PITCH + 8 * half];
        const uint16_t* ob_ = &sO[buf][col * PITCH + 8 * half];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          s = mfma32(lds_read_b128(qb_ + 16 * ks), kreg[ks], s);
          dp = mfma32(lds_read_b128(ob_ + 16 * ks), vreg[ks], dp);
        }
      }
      float lrow[16], drow[16];
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float4 l4 = *reinterpret_cast<const float4*>(&sL[buf][8 * q4 + 4 * half]);
        const float4 d4 = *reinterpret_cast<const float4*>(&sD[buf][8 * q4 + 4 * half]);
        lrow[4 * q4] = l4.x; lrow[4 * q4 + 1] = l4.y; lrow[4 * q4 + 2] = l4.z; lrow[4 * q4 + 3] = l4.w;
        drow[4 * q4] = d4.x; drow[4 * q4 + 1] = d4.y; drow[4 * q4 + 2] = d4.z; drow[4 * q4 + 3] = d4.w;
      }
      f32x16 p, ds;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = s[r] * a.scale_log2 - lrow[r];
        if (cls == kPartial) {
          const int i = i0 + 8 * (r >> 2) + 4 * half + (r & 3);
          const bool vis = (j <= i) && (i < ej) && (i < tr.L);
          if (!vis) x = -INFINITY;
        }
        p[r] = __builtin_amdgcn_exp2f(x);
        ds[r] = p[r] * (dp[r] - drow[r]);
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16x8 pb = pack8(p, 8 * t);
        const bf16x8 dsb = pack8(ds, 8 * t);
#pragma unroll
        for (int d = 0; d < DB; ++d) {
          dv[d] = mfma32(tr_operand<PITCH>(sO[buf], 16 * t, 32 * d, lane), pb, dv[d]);
          dk[d] = mfma32(tr_operand<PITCH>(sQ[buf], 16 * t, 32 * d, lane), dsb, dk[d]);
        }
      }
    }
    if (more) store(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  if (key_ok) {
    const size_t koff = ((size_t)(tr.tok0 + j) * a.Hkv + g) * D;
    const float sc = a.scale;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int dd = 32 * d + 8 * q4 + 4 * half;
        *reinterpret_cast<uint2*>(a.dk + koff + dd) =
            pack4_bf16(dk[d][4 * q4] * sc, dk[d][4 * q4 + 1] * sc, dk[d][4 * q4 + 2] * sc, dk[d][4 * q4 + 3] * sc);
        *reinterpret_cast<uint2*>(a.dv + koff + dd) =
            pack4_bf16(dv[d][4 * q4], dv[d][4 * q4 + 1], dv[d][4 * q4 + 2], dv[d][4 * q4 + 3]);
      }
  }
}

// ---------------------------------------------------------------- launchers
size_t ws_kstats_bytes(int B, int ntok) {
  const size_t n = (size_t)B + (size_t)ntok / kKeyTile + 2;
  return (n * sizeof(int2) + 255) & ~(size_t)255;
}

size_t ws_delta_bytes(int Hq, int ntok) { return ((size_t)Hq * ntok * sizeof(float) + 255) & ~(size_t)255; }

static RowArgs row_args(const Problem& p, const int2* kstats) {
  RowArgs a{};
  a.q = (const uint16_t*)p.q;
  a.k = (const uint16_t*)p.k;
  a.v = (const uint16_t*)p.v;
  a.evict = p.evict;
  a.cu = p.cu;
  a.kstats = kstats;
  a.o = (uint16_t*)p.o;
  a.lse = p.lse;
  a.dout = (const uint16_t*)p.dout;
  a.lse_in = p.lse_in;
  a.dq = (uint16_t*)p.dq;
  a.B = p.B;
  a.T = p.T;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.G = p.G;
  a.HG = p.HG;
  a.TC = p.TC;
  a.nhg = p.nhg;
  a.nqt = (p.T + 32 * p.TC - 1) / (32 * p.TC);
  a.ntok = p.ntok;
  a.varlen = p.cu != nullptr;
  a.scale = p.scale;
  a.scale_log2 = p.scale * 1.4426950408889634f;
  return a;
}

hipError_t launch_kstats(const Problem& p, int BN, int2* kstats) {
  dim3 grid(((p.T + BN - 1) / BN + kWave - 1) / kWave, p.B);
  prof_begin("classify", p.stream);
  hipLaunchKernelGGL(kstats_kernel, grid, dim3(kWave), 0, p.stream, p.evict, p.cu, p.T, BN, kstats);
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_fwd(const Problem& p, const int2* kstats) {
  RowArgs a = row_args(p, kstats);
  const long long nblk = (long long)a.nqt * p.B * p.Hkv * p.nhg;
  dim3 grid((unsigned)nblk), block(64 * p.HG * p.TC);
  prof_begin("fwd", p.stream);
  if (p.D == 128) hipLaunchKernelGGL(fwd_kernel<128>, grid, block, 0, p.stream, a);
  else hipLaunchKernelGGL(fwd_kernel<64>, grid, block, 0, p.stream, a);
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_bwd_pre(const Problem& p, float* delta) {
  const long long rows = (long long)p.ntok * p.Hq;
  dim3 grid((unsigned)((rows + 15) / 16)), block(256);
  prof_begin("bwd_pre", p.stream);
  if (p.D == 128)
    hipLaunchKernelGGL(bwd_pre_kernel<128>, grid, block, 0, p.stream, (const uint16_t*)p.o_in,
                       (const uint16_t*)p.dout, delta, p.ntok, p.Hq, p.T, (int)(p.cu != nullptr));
  else
    hipLaunchKernelGGL(bwd_pre_kernel<64>, grid, block, 0, p.stream, (const uint16_t*)p.o_in,
                       (const uint16_t*)p.dout, delta, p.ntok, p.Hq, p.T, (int)(p.cu != nullptr));
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const Problem& p, const float* delta) {
  ColArgs a{};
  a.q = (const uint16_t*)p.q;
  a.k = (const uint16_t*)p.k;
  a.v = (const uint16_t*)p.v;
  a.dout = (const uint16_t*)p.dout;
  a.lse = p.lse_in;
  a.delta = delta;
  a.evict = p.evict;
  a.cu = p.cu;
  a.dk = (uint16_t*)p.dk;
  a.dv = (uint16_t*)p.dv;
  a.B = p.B;
  a.T = p.T;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.G = p.G;
  a.nkt = (p.T + kColKeys - 1) / kColKeys;
  a.ntok = p.ntok;
  a.varlen = p.cu != nullptr;
  a.scale = p.scale;
  a.scale_log2 = p.scale * 1.4426950408889634f;
  const long long nblk = (long long)a.nkt * p.B * p.Hkv;
  prof_begin("bwd_dkdv", p.stream);
  if (p.D == 128) hipLaunchKernelGGL(dkdv_kernel<128>, dim3((unsigned)nblk), dim3(256), 0, p.stream, a);
  else hipLaunchKernelGGL(dkdv_kernel<64>, dim3((unsigned)nblk), dim3(256), 0, p.stream, a);
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const Problem& p, const int2* kstats, const float* delta) {
  RowArgs a = row_args(p, kstats);
  a.delta = delta;
  const long long nblk = (long long)a.nqt * p.B * p.Hkv * p.nhg;
  dim3 grid((unsigned)nblk), block(64 * p.HG * p.TC);
  prof_begin("bwd_dq", p.stream);
  if (p.D == 128) hipLaunchKernelGGL(dq_kernel<128>, grid, block, 0, p.stream, a);
  else hipLaunchKernelGGL(dq_kernel<64>, grid, block, 0, p.stream, a);
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_classify(const int32_t* evict, const int32_t* cu, int B, int T, int BM, int BN, uint8_t* out,
                           hipStream_t stream) {
  const int nk = (T + BN - 1) / BN, nq = (T + BM - 1) / BM;
  hipLaunchKernelGGL(classify_kernel, dim3((nk + kWave - 1) / kWave, nq, B), dim3(kWave), 0, stream, evict, cu, B,
                     T, BM, BN, out);
  return hipGetLastError();
}

hipError_t launch_check(const int32_t* evict, const int32_t* cu, int B, int T, int ntok, int64_t* first_bad,
                        int* cu_bad, hipStream_t stream) {
  hipLaunchKernelGGL(check_init_kernel, dim3(1), dim3(1), 0, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int blocks = (T + 255) / 256 < 1024 ? (T + 255) / 256 : 1024;
  hipLaunchKernelGGL(check_kernel, dim3(blocks > 0 ? blocks : 1, B), dim3(256), 0, stream, evict, cu, B, T, ntok);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  unsigned long long fb = 0;
  int cb = 0;
  e = hipMemcpyFromSymbolAsync(&fb, HIP_SYMBOL(g_first_bad), sizeof(fb), 0, hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  e = hipMemcpyFromSymbolAsync(&cb, HIP_SYMBOL(g_cu_bad), sizeof(cb), 0, hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return e;
  *first_bad = (fb == ULLONG_MAX) ? -1 : (int64_t)fb;
  *cu_bad = cb;
  return hipSuccess;
}

}  // namespace kvs
