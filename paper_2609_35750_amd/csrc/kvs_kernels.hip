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

#include <algorithm>
#include <climits>
#include <mutex>
#include <type_traits>

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
  int flags;            // kFlagNoEmptySkip | kFlagFullAsPartial (consistency checks; 0 normally)
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
  const int* plan;      // [B * nkt][2]: chunks of the key block (1 = not split), first slot
  const int2* items;    // [B * nkt + capE]: (key block, chunk) work items, longest first; (-1, 0) unused
  float* part;          // [capE * Hkv][2][kColKeys][D] fp32 partial dV, dK of split blocks
  int B, T, Hq, Hkv, G, nkt, ntok;
  int capE;             // slots per KV head (0: no splitting)
  int varlen;
  int flags;            // as in RowArgs
  float scale_log2;
  float scale;
};

// Row-step chunk of a split key block: 64 row-steps of 64 query rows; blocks
// whose span exceeds two chunks are split (see split_plan_kernel).
constexpr int kSplitRowSteps = 64;

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
                                                    int T, int ntok, int BN, int2* __restrict__ out) {
  const int kt = blockIdx.x * kWave + threadIdx.x, b = blockIdx.y;
  const Trace tr = trace_of(cu, b, T, ntok);
  const int j0 = kt * BN;
  if (j0 >= tr.L) return;
  out[kstat_index(b, tr.tok0, kt, BN)] = key_tile_stats(evict, tr, j0, BN);
}

// ---------------------------------------------------------------- tile-class grid
// One thread per (trace, q-tile, k-tile); grids of all traces concatenated.
// With cu_seqlens, T is the packed token count (every trace length is clamped
// to it, so the grids never outgrow what the host sized from the same offsets).
__global__ void __launch_bounds__(64) classify_kernel(const int* __restrict__ evict, const int* __restrict__ cu,
                                                      int B, int T, int BM, int BN, uint8_t* __restrict__ out) {
  const int kt = blockIdx.x * kWave + threadIdx.x;
  const int qt = blockIdx.y, b = blockIdx.z;
  const Trace tr = trace_of(cu, b, T, T);
  const int nq = (tr.L + BM - 1) / BM, nk = (tr.L + BN - 1) / BN;
  if (qt >= nq || kt >= nk) return;
  long long off = 0;
  for (int bb = 0; bb < b; ++bb) {
    const Trace t2 = trace_of(cu, bb, T, T);
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
  const Trace tr = trace_of(cu, b, T, ntok);
  if (tr.L <= 0) return;
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j < tr.L; j += gridDim.x * blockDim.x) {
    if (evict[tr.tok0 + j] <= j) atomicMin(&g_first_bad, (unsigned long long)(tr.tok0 + j));
  }
}

// ---------------------------------------------------------------- key-tile walker
// Every wave of a workgroup walks the same sequence of non-EMPTY key tiles of
// its query rows [i0, i1): 64 candidate tiles are classified at a time (one
// per lane) and the non-EMPTY ones kept as a ballot.  Each lane keeps the
// evict_at statistics of its candidate tile, so the statistics of the tile
// walker_next returns are read from a register (walker_stats) instead of from
// memory, whose latency the wave would otherwise wait out on every tile.
struct TileWalker {
  int base, lim;
  unsigned long long live;
  int emin, emax;   // statistics of candidate tile base + lane
};

__device__ __forceinline__ void walker_load(TileWalker& w, const int2* __restrict__ ks, int kidx0, int i0, int i1,
                                            int L, int flags) {
  const int kt = w.base + (threadIdx.x & 63);
  bool ne = false;
  int2 st = make_int2(0, 0);
  if (kt < w.lim) {
    st = ks[kidx0 + kt];
    ne = adjust_class(tile_class(i0, i1, kt * kKeyTile, kt * kKeyTile + kKeyTile, L, st.x, st.y), flags) != kEmpty;
  }
  w.live = __ballot(ne);
  w.emin = st.x;
  w.emax = st.y;
}

__device__ __forceinline__ int walker_next(TileWalker& w, const int2* __restrict__ ks, int kidx0, int i0, int i1,
                                           int L, int flags) {
  while (w.live == 0ull) {
    w.base += 64;
    if (w.base >= w.lim) return -1;
    walker_load(w, ks, kidx0, i0, i1, L, flags);
  }
  const int bit = __builtin_ctzll(w.live);
  w.live &= w.live - 1ull;
  return w.base + bit;
}

// evict_at minimum and maximum of tile kt, the tile the last walker_next call returned (kt >= 0)
__device__ __forceinline__ int2 walker_stats(const TileWalker& w, int kt) {
  const int l = kt - w.base;
  return make_int2(__builtin_amdgcn_readlane(w.emin, l), __builtin_amdgcn_readlane(w.emax, l));
}

// ---------------------------------------------------------------- operand reads from swizzled tiles
// S^T block (32 keys x 32 queries) of the current tile: A = K rows from LDS, B = Q^T in registers.
// rl = Lay<D, COMPACT>::row_lane(lane).
template <int D, bool COMPACT = false>
__device__ __forceinline__ f32x16 scores_t(const uint16_t* tile, int row0, const bf16x8* breg,
                                           typename Lay<D, COMPACT>::RowLane rl, f32x16 s = f32x16{}) {
  using LY = Lay<D, COMPACT>;
  const uint16_t* base = tile + row0 * LY::PITCH;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) s = mfma32(lds_read_b128(base + LY::row_at(rl, ks)), breg[ks], s);
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

// Head grouping of a row-kernel workgroup.
struct RowTile {
  int g, h, b, i0, i1, i0w, hh;
  Trace tr;
};

// Launch order: blockIdx % Hkv is the KV head (consecutive workgroups go to
// different XCDs, so each XCD's L2 serves one head's K/V); then the head
// group; then the traces one after another, each trace's query tiles from the
// last to the first (later tiles see more keys: start them first).  Taking
// the traces one at a time keeps an XCD's K/V working set to one trace.
__device__ __forceinline__ bool row_tile(const RowArgs& a, RowTile& t) {
  int wg = blockIdx.x;
  t.g = wg % a.Hkv;
  wg /= a.Hkv;
  const int hgrp = wg % a.nhg;
  wg /= a.nhg;
  const int qt = a.nqt - 1 - wg % a.nqt;
  t.b = wg / a.nqt;
  t.tr = trace_of(a.cu, t.b, a.T, a.ntok);
  const int BMt = 32 * a.TC;
  t.i0 = qt * BMt;
  t.i1 = t.i0 + BMt;
  if (t.i0 >= t.tr.L) return false;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  t.hh = wave % a.HG;
  t.h = t.g * a.G + hgrp * a.HG + t.hh;
  t.i0w = t.i0 + 32 * (wave / a.HG);
  return true;
}

// Asynchronous staging of one 64-key K/V (and evict_at) tile of KV head g
// (compact layout: two workgroups of the dQ kernel share a CU).
template <int D>
using KVStager = RowStager<D, kKeyTile, 4, true>;   // row kernels: 4 waves

template <int D>
__device__ __forceinline__ void stage_kv(const KVStager<D>& st, uint16_t* sK, uint16_t* sV, int* sE, const RowArgs& a,
                                         const RowTile& rt, int kt, int wave, int nw, int lane) {
  const int j0 = kt * kKeyTile;
  const long long base = ((long long)rt.tr.tok0 * a.Hkv + rt.g) * D;
  const long long stride = (long long)a.Hkv * D;
  st.issue(lds_addr(sK), a.k + base, stride, j0, rt.tr.L - 1, wave);
  st.issue(lds_addr(sV), a.v + base, stride, j0, rt.tr.L - 1, wave);
  if (wave == nw - 1) stage_words(lds_addr(sE), a.evict + rt.tr.tok0, j0, rt.tr.L - 1, lane);
}

// ---------------------------------------------------------------- forward
// K/V are staged in sub-tiles of BN keys (D = 128: 32, so that a workgroup
// needs 37 KB of LDS and three workgroups, three waves per SIMD, share a CU;
// D = 64: 64 keys, 37 KB, four workgroups at 128 VGPRs per wave), walked in
// the order of the non-EMPTY 64-key tiles.  The sub-tiles are double-buffered
// in two distinct LDS arrays each; the loop body alternates between them so
// the compiler can tell that the asynchronous fill of the next buffer never
// aliases the reads of the current one (and does not wait for the fill
// before reading).  A sub-tile's class comes from the statistics of its
// 64-key tile, which can only report PARTIAL where FULL would hold or
// non-EMPTY where EMPTY would: a conservative, exact choice.
template <int D>
constexpr int fwd_bn() { return D == 128 ? 32 : 64; }

template <int D>
using FwdStager = RowStager<D, fwd_bn<D>(), 4, true>;   // 4 waves

template <int D>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(D == 128 ? 3 : 4, D == 128 ? 3 : 4)))
fwd_kernel(RowArgs a) {
  constexpr int KS = D / 16, DB = D / 32, BN = fwd_bn<D>(), NKB = BN / 32, NSUB = kKeyTile / BN;
  __shared__ __attribute__((aligned(1024))) uint16_t sK0[BN * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sK1[BN * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sV0[BN * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sV1[BN * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(256))) int sE0[BN];
  __shared__ __attribute__((aligned(256))) int sE1[BN];

  RowTile rt;
  if (!row_tile(a, rt)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), nw = blockDim.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const Trace tr = rt.tr;
  const int i = rt.i0w + col;
  const bool row_ok = i < tr.L;
  const auto rl = Lay<D, true>::row_lane(lane);
  const int tl = Lay<D, true>::tr_lo(lane), th = Lay<D, true>::tr_hi(lane);
  FwdStager<D> kvst;
  kvst.init(wave, lane, (long long)a.Hkv * D);
  // asynchronous staging of sub-tile (kt, sub) of KV head g
  auto stage = [&](uint16_t* sK, uint16_t* sV, int* sE, int kt, int sub) __attribute__((always_inline)) {
    const int j0 = kt * kKeyTile + sub * BN;
    const long long base = ((long long)rt.tr.tok0 * a.Hkv + rt.g) * D;
    const long long stride = (long long)a.Hkv * D;
    kvst.issue(lds_addr(sK), a.k + base, stride, j0, rt.tr.L - 1, wave);
    kvst.issue(lds_addr(sV), a.v + base, stride, j0, rt.tr.L - 1, wave);
    if (wave == nw - 1) {
      if (BN == kWave || lane < BN) stage_words(lds_addr(sE), a.evict + rt.tr.tok0, j0, rt.tr.L - 1, lane);
    }
  };

  bf16x8 qreg[KS];
  {
    const uint16_t* qrow = a.q + ((size_t)(tr.tok0 + min(i, tr.L - 1)) * a.Hq + rt.h) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qreg[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qrow + 16 * ks));
  }

  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) acc[d] = f32x16{};
  // Running reference maximum of the row (log2 units), the offset the
  // exponentials use (0 until the row has seen a visible key), and the raw
  // score above which the reference must move: m_run + 8 in score units.
  float m_run = -INFINITY, l_run = 0.f, m_use = 0.f, thr = -INFINITY;
  const float inv_scale_log2 = 1.f / a.scale_log2;

  const int kidx0 = kstat_index(rt.b, tr.tok0, 0, kKeyTile);
  TileWalker w{0, (min(rt.i1, tr.L) + kKeyTile - 1) / kKeyTile, 0ull, 0, 0};
  walker_load(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L, a.flags);
  int kt = __builtin_amdgcn_readfirstlane(walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L, a.flags));
  int2 kst = kt >= 0 ? walker_stats(w, kt) : make_int2(0, 0);
  int sub = 0;

  // One tile: prefetch the next tile into (nK, nV, nE), compute on (cK, cV, cE).
  auto body = [&](const uint16_t* cK, const uint16_t* cV, const int* cE, uint16_t* nK, uint16_t* nV, int* nE) {
    // The next tile's statistics come from the walker's registers (no memory
    // access) and are used one iteration later.
    int nkt = kt, nsub = sub + 1;
    int2 nkst = kst;
    // next 64-key tile once this one is done or its remaining keys lie past the trace end
    // (a staged sub-tile must start inside the trace)
    if (nsub == NSUB || kt * kKeyTile + nsub * BN >= tr.L) {
      nkt = __builtin_amdgcn_readfirstlane(walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L, a.flags));
      nsub = 0;
      if (nkt >= 0) nkst = walker_stats(w, nkt);
    }
    if (nkt >= 0) stage(nK, nV, nE, nkt, nsub);
    const int j0 = kt * kKeyTile + sub * BN;
    const int cls = adjust_class(tile_class(rt.i0w, rt.i0w + 32, j0, j0 + BN, tr.L, kst.x, kst.y), a.flags);
    if (cls != kEmpty) {
      f32x16 s[NKB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        s[kb] = scores_t<D, true>(cK, 32 * kb, qreg, rl);
        if (cls == kPartial) mask_t(s[kb], cE, kb, j0, i, tr.L, half);
      }
      float mx = -INFINITY;   // maximum of this lane's half of the row
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
      // The reference max of a row only moves when the tile's max exceeds it by
      // more than 8 (log2 units): probabilities are then at most 2^8, exact to
      // rescale later, and the accumulator rescale is skipped for most tiles.
      // The row's max exceeds the threshold iff one of its two halves does, so
      // the halves are combined only when some row of the wave moves.  The
      // ballot moves every row of the wave, including rows that have not seen
      // a visible key yet and see none here (m_run = row max = -inf): their
      // factor is 1, not exp2(-inf - -inf) = NaN.
      if (__ballot(mx > thr)) {
        const float m_new = fmaxf(m_run, fmaxf(mx, wave_xor32(mx)) * a.scale_log2);
        const float alpha = m_new == m_run ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);   // 0 on the first visible tile
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[d][r] *= alpha;
        m_run = m_new;
        m_use = (m_run == -INFINITY) ? 0.f : m_run;
        thr = (m_run + 8.f) * inv_scale_log2;
      }
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][r], a.scale_log2, -m_use));
          s[kb][r] = p;
          ls += p;
        }
      l_run += ls;
      // Raised wave priority for the PV products: the SIMD then runs this wave's
      // MFMAs back to back while the other resident waves do their softmax work,
      // instead of the waves drifting into the same phase (measured: 2-3%).
      __builtin_amdgcn_s_setprio(3);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8 pb = pack8(s[kb], 8 * t);
#pragma unroll
          for (int d = 0; d < DB; ++d)
            acc[d] = mfma32(tr_operand<D, true>(cV, 32 * kb + 16 * t, 32 * d, tl, th), pb, acc[d]);
        }
      __builtin_amdgcn_s_setprio(0);
    }
    wait_vm();
    __syncthreads();
    kt = nkt;
    sub = nsub;
    kst = nkst;
  };

  if (kt >= 0) stage(sK0, sV0, sE0, kt, 0);
  wait_vm();
  __syncthreads();
  while (kt >= 0) {
    body(sK0, sV0, sE0, sK1, sV1, sE1);
    if (kt < 0) break;
    body(sK1, sV1, sE1, sK0, sV0, sE0);
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

// ---------------------------------------------------------------- backward: Delta = rowsum(dO * O), stored as -Delta
// Also writes LSE * log2(e), the form in which the backward kernels use it.
template <int D>
__global__ void __launch_bounds__(256) bwd_pre_kernel(const uint16_t* __restrict__ o, const uint16_t* __restrict__ dout,
                                                      const float* __restrict__ lse, float* __restrict__ delta,
                                                      float* __restrict__ lse2, int ntok, int Hq, int T, int varlen) {
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
    delta[idx] = -s;   // stored negated: both backward kernels add it
    lse2[idx] = lse[idx] * 1.4426950408889634f;
  }
}

// ---------------------------------------------------------------- backward: dQ (row kernel)
template <int D>
__global__ void __launch_bounds__(512) dq_kernel(RowArgs a) {
  constexpr int KS = D / 16, DB = D / 32;
  __shared__ __attribute__((aligned(1024))) uint16_t sK0[kKeyTile * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sK1[kKeyTile * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sV0[kKeyTile * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sV1[kKeyTile * Lay<D, true>::PITCH];
  __shared__ __attribute__((aligned(256))) int sE0[kKeyTile];
  __shared__ __attribute__((aligned(256))) int sE1[kKeyTile];

  RowTile rt;
  if (!row_tile(a, rt)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), nw = blockDim.x >> 6;
  const int half = lane >> 5, col = lane & 31;
  const Trace tr = rt.tr;
  const int i = rt.i0w + col;
  const bool row_ok = i < tr.L;
  const auto rl = Lay<D, true>::row_lane(lane);
  const int tl = Lay<D, true>::tr_lo(lane), th = Lay<D, true>::tr_hi(lane);
  KVStager<D> kvst;
  kvst.init(wave, lane, (long long)a.Hkv * D);
  const int ic = min(i, tr.L - 1);

  bf16x8 qreg[KS], oreg[KS];
  float lse2, ndlt;
  {
    const size_t roff = ((size_t)(tr.tok0 + ic) * a.Hq + rt.h) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qreg[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(a.q + roff + 16 * ks));
      oreg[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(a.dout + roff + 16 * ks));
    }
    const long long li = lse_index(a.varlen, a.ntok, a.Hq, a.T, rt.b, rt.h, tr.tok0, ic);
    lse2 = a.lse_in[li];   // already scaled by log2(e)
    ndlt = a.delta[li];   // -Delta
  }

  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) acc[d] = f32x16{};

  const int kidx0 = kstat_index(rt.b, tr.tok0, 0, kKeyTile);
  TileWalker w{0, (min(rt.i1, tr.L) + kKeyTile - 1) / kKeyTile, 0ull, 0, 0};
  walker_load(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L, a.flags);
  int kt = __builtin_amdgcn_readfirstlane(walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L, a.flags));
  int2 kst = kt >= 0 ? walker_stats(w, kt) : make_int2(0, 0);

  auto body = [&](const uint16_t* cK, const uint16_t* cV, const int* cE, uint16_t* nK, uint16_t* nV, int* nE) {
    // The next tile's statistics come from the walker's registers (no memory
    // access) and are used one iteration later.
    const int nkt = __builtin_amdgcn_readfirstlane(walker_next(w, a.kstats, kidx0, rt.i0, rt.i1, tr.L, a.flags));
    int2 nkst = make_int2(0, 0);
    if (nkt >= 0) {
      nkst = walker_stats(w, nkt);
      stage_kv<D>(kvst, nK, nV, nE, a, rt, nkt, wave, nw, lane);
    }
    const int j0 = kt * kKeyTile;
    const int cls = adjust_class(tile_class(rt.i0w, rt.i0w + 32, j0, j0 + kKeyTile, tr.L, kst.x, kst.y), a.flags);
    if (cls != kEmpty) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = scores_t<D, true>(cK, 32 * kb, qreg, rl);
        if (cls == kPartial) mask_t(s, cE, kb, j0, i, tr.L, half);
        // dP - Delta: the product starts at -Delta
        f32x16 d0;
#pragma unroll
        for (int r = 0; r < 16; ++r) d0[r] = ndlt;
        const f32x16 dp = scores_t<D, true>(cV, 32 * kb, oreg, rl, d0);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], a.scale_log2, -lse2));
          s[r] = p * dp[r];
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8 dsb = pack8(s, 8 * t);
#pragma unroll
          for (int d = 0; d < DB; ++d)
            acc[d] = mfma32(tr_operand<D, true>(cK, 32 * kb + 16 * t, 32 * d, tl, th), dsb, acc[d]);
        }
      }
    }
    wait_vm();
    __syncthreads();
    kt = nkt;
    kst = nkst;
  };

  if (kt >= 0) stage_kv<D>(kvst, sK0, sV0, sE0, a, rt, kt, wave, nw, lane);
  wait_vm();
  __syncthreads();
  while (kt >= 0) {
    body(sK0, sV0, sE0, sK1, sV1, sE1);
    if (kt < 0) break;
    body(sK1, sV1, sE1, sK0, sV0, sE0);
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
// One workgroup: 128 keys of one KV head, 8 waves.  Wave w < 4 (the "dV
// wave") and wave w + 4 (the "dK wave") own the same 32 keys and share a SIMD.
// The workgroup walks the query rows that can see any of its keys in steps of
// 64 rows x one q-head of the group; Q, dO, LSE and Delta of a step are staged
// once in LDS for all eight waves.  Per 32-row block:
//   dV wave:  S = Q K^T,  P = exp2(S * scale * log2 e - LSE * log2 e) (masked),
//             P -> LDS (bf16),  dV^T += dO^T P
//   dK wave:  dP = dO V^T - Delta,  dS = P dP  (P read back from LDS),
//             dK^T += Q^T dS
// The dV waves run one step ahead of the dK waves (P of step s is written
// during step s - 1), so a single barrier per step orders the exchange, every
// product is computed once, and the two waves of a SIMD issue the same number
// of MFMAs.  Masking happens only in the dV wave (masked P = 0 gives dS = 0).
template <int D>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) dkdv_kernel(ColArgs a) {
  constexpr int KS = D / 16, DB = D / 32, PITCH = Lay<D>::PITCH;
  __shared__ __attribute__((aligned(1024))) uint16_t sQ0[kQStep * PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sQ1[kQStep * PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sQ2[kQStep * PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sO0[kQStep * PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sO1[kQStep * PITCH];
  __shared__ __attribute__((aligned(1024))) uint16_t sO2[kQStep * PITCH];
  __shared__ __attribute__((aligned(256))) float sL0[kQStep];
  __shared__ __attribute__((aligned(256))) float sL1[kQStep];
  __shared__ __attribute__((aligned(256))) float sL2[kQStep];
  __shared__ __attribute__((aligned(256))) float sD0[kQStep];
  __shared__ __attribute__((aligned(256))) float sD1[kQStep];
  __shared__ __attribute__((aligned(256))) float sD2[kQStep];
  // P exchange: [step parity][key quarter][32-row block][half of the 16 values][lane], 8 fp16 each
  // (P <= 1; fp16 keeps 3 more mantissa bits than bf16 for dS = P dP)
  __shared__ __attribute__((aligned(1024))) f16x8 sP[2 * 4 * 2 * 2 * kWave];
  __shared__ int sEmax[4];

  // Work item of this workgroup (longest first, see split_plan_kernel): a
  // whole key block, or one row chunk of a split block; one KV head each.
  const int g = blockIdx.x % a.Hkv;
  const int2 item = a.items[blockIdx.x / a.Hkv];
  if (item.x < 0) return;   // unused list entry
  const int b = item.x / a.nkt, kt = item.x % a.nkt, chunk = item.y;
  const int nchunk = a.plan[2 * item.x], slot0 = a.plan[2 * item.x + 1];
  const Trace tr = trace_of(a.cu, b, a.T, a.ntok);
  const int j0 = kt * kColKeys;
  if (j0 >= tr.L) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool role_dk = wave >= 4;
  const int kw = wave & 3;
  const int half = lane >> 5, col = lane & 31;
  const int j = j0 + 32 * kw + col;
  const bool key_ok = j < tr.L;
  const int jc = min(j, tr.L - 1);
  const int ej = key_ok ? min(a.evict[tr.tok0 + j], tr.L) : 0;
  const unsigned kspan = key_ok ? (unsigned)(ej - j) : 0u;   // rows j .. ej - 1 see this key
  const auto rl = Lay<D>::row_lane(lane);
  const int tl = Lay<D>::tr_lo(lane), th = Lay<D>::tr_hi(lane);
  int emin_w = key_ok ? ej : INT_MAX, emax_w = key_ok ? ej : INT_MIN;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    emin_w = min(emin_w, __shfl_xor(emin_w, off));
    emax_w = max(emax_w, __shfl_xor(emax_w, off));
  }
  if (!role_dk && lane == 0) sEmax[kw] = emax_w;
  RowStager<D, kQStep, 8> qst;
  qst.init(wave, lane, (long long)a.Hq * D);

  // K (dV waves) or V (dK waves) of this lane's key: the B operand of S or dP
  bf16x8 kvreg[KS];
  {
    const size_t koff = ((size_t)(tr.tok0 + jc) * a.Hkv + g) * D + 8 * half;
    const uint16_t* src = role_dk ? a.v : a.k;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kvreg[ks] = as_bf16x8(*reinterpret_cast<const uint4*>(src + koff + 16 * ks));
  }
  __syncthreads();
  const int emax_wg = max(max(sEmax[0], sEmax[1]), max(sEmax[2], sEmax[3]));
  int qs_lo = j0 / kQStep;
  int qs_hi = (emax_wg + kQStep - 1) / kQStep;
  if (nchunk > 1) {
    qs_lo += chunk * kSplitRowSteps;
    qs_hi = min(qs_hi, qs_lo + kSplitRowSteps);
  }
  const int steps = max(qs_hi - qs_lo, 0) * a.G;

  f32x16 acc[DB];   // dV^T (dV waves) or dK^T (dK waves): rows d, column = this lane's key
#pragma unroll
  for (int d = 0; d < DB; ++d) acc[d] = f32x16{};

  auto stage = [&](uint16_t* q_, uint16_t* o_, float* l_, float* d_, int step) __attribute__((always_inline)) {
    const int i0 = (qs_lo + step / a.G) * kQStep;
    const int h = g * a.G + step % a.G;
    const long long base = ((long long)tr.tok0 * a.Hq + h) * D;
    qst.issue(lds_addr(q_), a.q + base, (long long)a.Hq * D, i0, tr.L - 1, wave);
    qst.issue(lds_addr(o_), a.dout + base, (long long)a.Hq * D, i0, tr.L - 1, wave);
    const long long lb = lse_index(a.varlen, a.ntok, a.Hq, a.T, b, h, tr.tok0, 0);
    if (wave == 6) stage_words(lds_addr(l_), a.lse + lb, i0, tr.L - 1, lane);   // LSE * log2(e)
    if (wave == 7) stage_words(lds_addr(d_), a.delta + lb, i0, tr.L - 1, lane);
  };
  const int jw0 = j0 + 32 * kw;
  auto xslot = [&](int step, int blk, int t) __attribute__((always_inline)) { return sP + ((((step & 1) * 4 + kw) * 2 + blk) * 2 + t) * kWave + lane; };

  // acc += (dO^T or Q^T) x for one 32-row block (A operand read transposed from the staged tile)
  auto block_acc = [&](const uint16_t* src, int rb, const bf16x8 (&xb)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int d = 0; d < DB; ++d) acc[d] = mfma32(tr_operand<D>(src, rb + 16 * t, 32 * d, tl, th), xb[t], acc[d]);
  };
  // dV wave, one 32-row block: S = Q K^T (C layout: lane <-> key, element r <->
  // row rb + 8 (r/4) + 4 half + r%4 of the staged tile), P, P -> LDS, dV^T += dO^T P.
  auto dv_block_s = [&](const uint16_t* cQ, const float* cL, int rb, int ib, bool partial, bf16x8 (&pb)[2],
                        f16x8 (&ph)[2]) __attribute__((always_inline)) {
    f32x16 x = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) x = mfma32(lds_read_b128(cQ + rb * PITCH + Lay<D>::row_at(rl, ks)), kvreg[ks], x);
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const float4 l4 = *reinterpret_cast<const float4*>(cL + rb + 8 * q4 + 4 * half);
      const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) x[4 * q4 + t] = __builtin_fmaf(x[4 * q4 + t], a.scale_log2, -lv[t]);
    }
    if (partial) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const bool vis = (unsigned)(ib + 8 * (r >> 2) + 4 * half + (r & 3) - j) < kspan;
        x[r] = vis ? x[r] : -INFINITY;
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = __builtin_amdgcn_exp2f(x[r]);
    pb[0] = pack8(x, 0);
    pb[1] = pack8(x, 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ph[0][e] = (_Float16)x[e];
      ph[1][e] = (_Float16)x[8 + e];
    }
  };
  // dK wave, one 32-row block: dP = dO V^T - Delta, dS = P dP with P from LDS.
  auto dk_block_s = [&](const uint16_t* cO, const float* cD, int rb, const f16x8* xp0, const f16x8* xp1,
                        bf16x8 (&sb)[2]) __attribute__((always_inline)) {
    f32x16 dp;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const float4 d4 = *reinterpret_cast<const float4*>(cD + rb + 8 * q4 + 4 * half);
      dp[4 * q4] = d4.x;   // -Delta
      dp[4 * q4 + 1] = d4.y;
      dp[4 * q4 + 2] = d4.z;
      dp[4 * q4 + 3] = d4.w;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) dp = mfma32(lds_read_b128(cO + rb * PITCH + Lay<D>::row_at(rl, ks)), kvreg[ks], dp);
    const f16x8 p0 = *xp0, p1 = *xp1;
    f32x16 x;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      x[e] = (float)p0[e] * dp[e];
      x[8 + e] = (float)p1[e] * dp[8 + e];
    }
    sb[0] = pack8(x, 0);
    sb[1] = pack8(x, 8);
  };

  // Both 32-row blocks FULL (the common case), written as one straight-line
  // sequence whose order is pinned with scheduling fences: all LDS operands of
  // the score products are requested before the first product, and the
  // transposed operands of each accumulation are requested while the
  // exponentials of that block are computed, so LDS latency overlaps work.
  auto dv_full = [&](int step, const uint16_t* cQ, const uint16_t* cO, const float* cL) __attribute__((always_inline)) {
    bf16x8 qa[2][KS];
    float4 lv[2][4];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qa[blk][ks] = lds_read_b128(cQ + 32 * blk * PITCH + Lay<D>::row_at(rl, ks));
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) lv[blk][q4] = *reinterpret_cast<const float4*>(cL + 32 * blk + 8 * q4 + 4 * half);
    }
    __builtin_amdgcn_sched_barrier(0);
    f32x16 x[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      x[blk] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) x[blk] = mfma32(qa[blk][ks], kvreg[ks], x[blk]);
    }
    bf16x8 tA[2][DB], tB[2][DB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int d = 0; d < DB; ++d) tA[t][d] = tr_operand<D>(cO, 16 * t, 32 * d, tl, th);
    __builtin_amdgcn_sched_barrier(0);
    bf16x8 pb[2][2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const float lq[4] = {lv[blk][q4].x, lv[blk][q4].y, lv[blk][q4].z, lv[blk][q4].w};
#pragma unroll
        for (int t = 0; t < 4; ++t)
          x[blk][4 * q4 + t] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[blk][4 * q4 + t], a.scale_log2, -lq[t]));
      }
      pb[blk][0] = pack8(x[blk], 0);
      pb[blk][1] = pack8(x[blk], 8);
      f16x8 h0, h1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        h0[e] = (_Float16)x[blk][e];
        h1[e] = (_Float16)x[blk][8 + e];
      }
      *xslot(step, blk, 0) = h0;
      *xslot(step, blk, 1) = h1;
      if (blk == 0) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int d = 0; d < DB; ++d) tB[t][d] = tr_operand<D>(cO, 32 + 16 * t, 32 * d, tl, th);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int d = 0; d < DB; ++d) acc[d] = mfma32(tA[t][d], pb[0][t], acc[d]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int d = 0; d < DB; ++d) acc[d] = mfma32(tB[t][d], pb[1][t], acc[d]);
  };
  auto dk_full = [&](int step, const uint16_t* cQ, const uint16_t* cO, const float* cD) __attribute__((always_inline)) {
    bf16x8 oa[2][KS];
    f32x16 dp[2];
    f16x8 pr[2][2];
    float4 dv4[2][4];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) oa[blk][ks] = lds_read_b128(cO + 32 * blk * PITCH + Lay<D>::row_at(rl, ks));
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) dv4[blk][q4] = *reinterpret_cast<const float4*>(cD + 32 * blk + 8 * q4 + 4 * half);
      pr[blk][0] = *xslot(step, blk, 0);
      pr[blk][1] = *xslot(step, blk, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {   // start at -Delta, so the product gives dP - Delta
        dp[blk][4 * q4] = dv4[blk][q4].x;
        dp[blk][4 * q4 + 1] = dv4[blk][q4].y;
        dp[blk][4 * q4 + 2] = dv4[blk][q4].z;
        dp[blk][4 * q4 + 3] = dv4[blk][q4].w;
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) dp[blk] = mfma32(oa[blk][ks], kvreg[ks], dp[blk]);
    }
    bf16x8 tA[2][DB], tB[2][DB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int d = 0; d < DB; ++d) tA[t][d] = tr_operand<D>(cQ, 16 * t, 32 * d, tl, th);
    __builtin_amdgcn_sched_barrier(0);
    bf16x8 sb[2][2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      f32x16 x;
#pragma unroll
      for (int r = 0; r < 16; ++r) x[r] = (float)pr[blk][r >> 3][r & 7] * dp[blk][r];
      sb[blk][0] = pack8(x, 0);
      sb[blk][1] = pack8(x, 8);
      if (blk == 0) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int d = 0; d < DB; ++d) tB[t][d] = tr_operand<D>(cQ, 32 + 16 * t, 32 * d, tl, th);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int d = 0; d < DB; ++d) acc[d] = mfma32(tA[t][d], sb[0][t], acc[d]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int d = 0; d < DB; ++d) acc[d] = mfma32(tB[t][d], sb[1][t], acc[d]);
  };
  auto dv_step = [&](int step, const uint16_t* cQ, const uint16_t* cO, const float* cL) __attribute__((always_inline)) {
    const int i0 = (qs_lo + step / a.G) * kQStep;
    const int c0 = adjust_class(tile_class(i0, i0 + 32, jw0, jw0 + 32, tr.L, emin_w, emax_w), a.flags);
    const int c1 = adjust_class(tile_class(i0 + 32, i0 + 64, jw0, jw0 + 32, tr.L, emin_w, emax_w), a.flags);
    if (c0 == kFull && c1 == kFull) {
      dv_full(step, cQ, cO, cL);
    } else {
      if (c0 != kEmpty) {
        bf16x8 p0[2];
        f16x8 h0[2];
        dv_block_s(cQ, cL, 0, i0, c0 == kPartial, p0, h0);
        *xslot(step, 0, 0) = h0[0];
        *xslot(step, 0, 1) = h0[1];
        block_acc(cO, 0, p0);
      }
      if (c1 != kEmpty) {
        bf16x8 p1[2];
        f16x8 h1[2];
        dv_block_s(cQ, cL, 32, i0 + 32, c1 == kPartial, p1, h1);
        *xslot(step, 1, 0) = h1[0];
        *xslot(step, 1, 1) = h1[1];
        block_acc(cO, 32, p1);
      }
    }
  };
  auto dk_step = [&](int step, const uint16_t* cQ, const uint16_t* cO, const float* cD) __attribute__((always_inline)) {
    const int i0 = (qs_lo + step / a.G) * kQStep;
    const int c0 = adjust_class(tile_class(i0, i0 + 32, jw0, jw0 + 32, tr.L, emin_w, emax_w), a.flags);
    const int c1 = adjust_class(tile_class(i0 + 32, i0 + 64, jw0, jw0 + 32, tr.L, emin_w, emax_w), a.flags);
    if (c0 != kEmpty && c1 != kEmpty) {
      dk_full(step, cQ, cO, cD);
    } else {
      if (c0 != kEmpty) {
        bf16x8 s0[2];
        dk_block_s(cO, cD, 0, xslot(step, 0, 0), xslot(step, 0, 1), s0);
        block_acc(cQ, 0, s0);
      }
      if (c1 != kEmpty) {
        bf16x8 s1[2];
        dk_block_s(cO, cD, 32, xslot(step, 1, 0), xslot(step, 1, 1), s1);
        block_acc(cQ, 32, s1);
      }
    }
  };

  // Three-stage ring: during step s the dK waves read tile s, the dV waves tile
  // s + 1, and tile s + 2 is copied into the buffer tile s - 1 used.
  auto run = [&](auto dk_tag) __attribute__((always_inline)) {
    constexpr bool DK = decltype(dk_tag)::value;
    int step = 0;
    auto body = [&](const uint16_t* cQ, const uint16_t* cO, const float* cD, const uint16_t* nQ, const uint16_t* nO,
                    const float* nL, uint16_t* zQ, uint16_t* zO, float* zL, float* zD) __attribute__((always_inline)) {
      if (step + 2 < steps) stage(zQ, zO, zL, zD, step + 2);
      if (DK) dk_step(step, cQ, cO, cD);
      else if (step + 1 < steps) dv_step(step + 1, nQ, nO, nL);
      wait_vm();   // tile step + 2 has landed (the dV waves read it next step)
      __syncthreads();
      ++step;
    };
    if (steps > 0) stage(sQ0, sO0, sL0, sD0, 0);
    if (steps > 1) stage(sQ1, sO1, sL1, sD1, 1);
    wait_vm();
    __syncthreads();
    if (!DK && steps > 0) dv_step(0, sQ0, sO0, sL0);
    __syncthreads();
    while (step < steps) {
      body(sQ0, sO0, sD0, sQ1, sO1, sL1, sQ2, sO2, sL2, sD2);
      if (step >= steps) break;
      body(sQ1, sO1, sD1, sQ2, sO2, sL2, sQ0, sO0, sL0, sD0);
      if (step >= steps) break;
      body(sQ2, sO2, sD2, sQ0, sO0, sL0, sQ1, sO1, sL1, sD1);
    }
  };
  if (role_dk) run(std::true_type{});
  else run(std::false_type{});

  if (nchunk > 1) {
    // fp32 partial sums of this chunk: [slot][dV, dK][key in block][d]
    float* dst = a.part + (((size_t)(slot0 + chunk) * a.Hkv + g) * 2 + (role_dk ? 1 : 0)) * kColKeys * D +
                 (size_t)(32 * kw + col) * D;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<float4*>(dst + 32 * d + 8 * q4 + 4 * half) =
            make_float4(acc[d][4 * q4], acc[d][4 * q4 + 1], acc[d][4 * q4 + 2], acc[d][4 * q4 + 3]);
  } else if (key_ok) {
    const size_t koff = ((size_t)(tr.tok0 + j) * a.Hkv + g) * D;
    uint16_t* dst = role_dk ? a.dk + koff : a.dv + koff;
    const float sc = role_dk ? a.scale : 1.f;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<uint2*>(dst + 32 * d + 8 * q4 + 4 * half) =
            pack4_bf16(acc[d][4 * q4] * sc, acc[d][4 * q4 + 1] * sc, acc[d][4 * q4 + 2] * sc, acc[d][4 * q4 + 3] * sc);
  }
}

// ---------------------------------------------------------------- work plan of the column kernel
// A key block whose keys stay visible for many query rows (the prompt,
// long-lived summaries) would be one long workgroup and set the kernel's
// critical path.  Blocks spanning more than 2 * kSplitRowSteps row-steps are
// cut into chunks of kSplitRowSteps row-steps; every chunk gets a slot of fp32
// partial sums, and the chunks are added in slot order afterwards
// (deterministic).  Slots are granted in key-block order while capE lasts;
// later blocks stay whole.  All work items (whole blocks and chunks) are then
// listed longest first (counting sort on the row-step count), so the longest
// items start first.  One workgroup of 1024 threads; block spans come from the
// 64-key tile statistics.
__global__ void __launch_bounds__(1024) split_plan_kernel(const int2* __restrict__ kstats, const int* __restrict__ cu,
                                                          int B, int T, int ntok, int nkt, int capE,
                                                          int* __restrict__ plan, int2* __restrict__ items) {
  constexpr int NBK = 2048;   // sort buckets: row-step counts 0 .. 2047 (longer ones share the last bucket)
  __shared__ int scan[1024];
  __shared__ int bucket[NBK];
  const int tid = threadIdx.x;
  const int nblocks = B * nkt, nitems = nblocks + capE;
  for (int i = tid; i < NBK; i += 1024) bucket[i] = 0;
  for (int e = tid; e < nitems; e += 1024) items[e] = make_int2(-1, 0);
  const int per = (nblocks + 1023) / 1024;
  const int b0 = min(tid * per, nblocks), b1 = min(b0 + per, nblocks);
  auto span_of = [&](int blk) {   // query row-steps [j0/64, ceil(emax/64)) of the block; 0 past the trace
    const int b = blk / nkt, kt = blk % nkt;
    const Trace tr = trace_of(cu, b, T, ntok);
    const int j0 = kt * kColKeys;
    if (j0 >= tr.L) return 0;
    const int t0 = j0 / kKeyTile, nt = (tr.L + kKeyTile - 1) / kKeyTile;
    int emax = kstats[kstat_index(b, tr.tok0, t0, kKeyTile)].y;
    if (t0 + 1 < nt) emax = max(emax, kstats[kstat_index(b, tr.tok0, t0 + 1, kKeyTile)].y);
    return (emax + kQStep - 1) / kQStep - j0 / kQStep;
  };
  auto chunks_of = [](int span) {
    return span > 2 * kSplitRowSteps ? (span + kSplitRowSteps - 1) / kSplitRowSteps : 0;
  };
  // Sort key (larger first).  One trace (or more than NBK / 8): the row-step
  // count.  Otherwise the row-step count in classes of Q >= 8 steps, then the
  // trace, so that items of one trace with about the same length are listed
  // together and run side by side (they share Q / dO rows in an XCD's L2);
  // the longest class still starts first, so the tail grows by less than Q
  // steps.  Keys stay below NBK: nclass * B <= NBK.
  const bool by_trace = B > 1 && B <= NBK / 8;
  const int Q = by_trace ? max(8, (NBK + NBK / B - 1) / (NBK / B)) : 1;
  const int nclass = (NBK + Q - 1) / Q;
  auto key_of = [&](int rows, int blk) {
    const int r = min(rows, NBK - 1);
    return by_trace ? min(r / Q, nclass - 1) * B + blk / nkt : r;
  };
  int tot = 0;
  for (int blk = b0; blk < b1; ++blk) tot += chunks_of(span_of(blk));
  scan[tid] = tot;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int v = tid >= off ? scan[tid - off] : 0;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  int run = scan[tid] - tot;   // exclusive prefix of requested slots
  for (int blk = b0; blk < b1; ++blk) {
    const int span = span_of(blk), w = chunks_of(span);
    const bool grant = w > 0 && run + w <= capE;
    plan[2 * blk] = grant ? w : 1;
    plan[2 * blk + 1] = grant ? run : 0;
    run += w;
    if (span == 0) continue;
    if (grant)
      for (int c = 0; c < w; ++c) atomicAdd(&bucket[key_of(min(kSplitRowSteps, span - c * kSplitRowSteps), blk)], 1);
    else
      atomicAdd(&bucket[key_of(span, blk)], 1);
  }
  __syncthreads();
  // bucket start positions, longest first: thread t owns buckets NBK-1-2t and NBK-2-2t
  const int khi = NBK - 1 - 2 * tid, klo = khi - 1;
  const int chi = bucket[khi], clo = bucket[klo];
  scan[tid] = chi + clo;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int v = tid >= off ? scan[tid - off] : 0;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  const int excl = scan[tid] - chi - clo;
  bucket[khi] = excl;
  bucket[klo] = excl + chi;
  __syncthreads();
  for (int blk = b0; blk < b1; ++blk) {
    const int span = span_of(blk);
    if (span == 0) continue;
    const int nc = plan[2 * blk];
    if (nc > 1) {
      for (int c = 0; c < nc; ++c)
        items[atomicAdd(&bucket[key_of(min(kSplitRowSteps, span - c * kSplitRowSteps), blk)], 1)] = make_int2(blk, c);
    } else {
      items[atomicAdd(&bucket[key_of(span, blk)], 1)] = make_int2(blk, 0);
    }
  }
}

// Sum of the chunk partials of split key blocks, in chunk order; dK scaled.
// kReduceSplit workgroups per (key block, KV head), each summing a slice of
// the block's keys; blocks that were not split exit.
constexpr int kReduceSplit = 8;
template <int D>
__global__ void __launch_bounds__(256) split_reduce_kernel(const int* __restrict__ plan, const float* __restrict__ part,
                                                           const int* __restrict__ cu, uint16_t* __restrict__ dk,
                                                           uint16_t* __restrict__ dv, int B, int T, int ntok,
                                                           int nkt, int Hkv, float scale) {
  const int sub = blockIdx.x % kReduceSplit, wg = blockIdx.x / kReduceSplit;
  const int g = wg % Hkv, blk = wg / Hkv;
  const int nc = plan[2 * blk], s0 = plan[2 * blk + 1];
  if (nc <= 1) return;
  const int b = blk / nkt, kt = blk % nkt;
  const Trace tr = trace_of(cu, b, T, ntok);
  constexpr int PER = kColKeys * D / kReduceSplit / 256;   // elements per thread
  static_assert(PER % 4 == 0 && PER >= 4, "reduce slice must be whole float4s per thread");
  for (int which = 0; which < 2; ++which) {
    for (int q = 0; q < PER / 4; ++q) {
      const int e = sub * (kColKeys * D / kReduceSplit) + (q * 256 + threadIdx.x) * 4;   // element of [key][d]
      const int key = e / D, d = e % D;
      float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int c = 0; c < nc; ++c) {
        const float4 v = *reinterpret_cast<const float4*>(part + (((size_t)(s0 + c) * Hkv + g) * 2 + which) * kColKeys * D + e);
        sum.x += v.x;
        sum.y += v.y;
        sum.z += v.z;
        sum.w += v.w;
      }
      const int j = kt * kColKeys + key;
      if (j < tr.L) {
        const float sc = which ? scale : 1.f;
        uint16_t* dst = (which ? dk : dv) + ((size_t)(tr.tok0 + j) * Hkv + g) * D + d;
        *reinterpret_cast<uint2*>(dst) = pack4_bf16(sum.x * sc, sum.y * sc, sum.z * sc, sum.w * sc);
      }
    }
  }
}

// Explicit instantiations: every kernel the launchers use is emitted, with its host stub.
template __global__ void fwd_kernel<64>(RowArgs);
template __global__ void fwd_kernel<128>(RowArgs);
template __global__ void dq_kernel<64>(RowArgs);
template __global__ void dq_kernel<128>(RowArgs);
template __global__ void dkdv_kernel<64>(ColArgs);
template __global__ void dkdv_kernel<128>(ColArgs);
template __global__ void split_reduce_kernel<64>(const int*, const float*, const int*, uint16_t*, uint16_t*, int, int,
                                                 int, int, int, float);
template __global__ void split_reduce_kernel<128>(const int*, const float*, const int*, uint16_t*, uint16_t*, int, int,
                                                  int, int, int, float);

// ---------------------------------------------------------------- library-owned scratch (allocation-free forward)
// Per-key-tile statistics of kvs_evict_attn_fwd_noalloc.  In host code the
// name `scratch` is only a host-side stand-in: its device address (one per
// GPU) comes from hipGetSymbolAddress, taken once per device with that device
// current, and only that address is ever passed to a kernel.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

hipError_t noalloc_scratch(void** ptr) {
  static std::mutex mu;
  static void* per_device[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!per_device[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    per_device[dev] = p;
  }
  *ptr = per_device[dev];
  return hipSuccess;
}

// ---------------------------------------------------------------- launchers
size_t ws_kstats_bytes(int B, int ntok) {
  const size_t n = (size_t)B + (size_t)ntok / kKeyTile + 2;
  return (n * sizeof(int2) + 255) & ~(size_t)255;
}

// -Delta followed by LSE * log2(e), each [Hq][ntok] (or [B][Hq][T]) fp32.
size_t ws_delta_bytes(int Hq, int ntok) { return 2 * (((size_t)Hq * ntok * sizeof(float) + 255) & ~(size_t)255); }

static size_t round256(size_t n) { return (n + 255) & ~(size_t)255; }

// Work plan of the column kernel: plan [B * nkt][2] int, work items
// [B * nkt + capE] int2, partial sums [capE * Hkv][2][kColKeys][D] fp32.
// capE: chunk slots per KV head, at most 2048 slots over all KV heads, none
// when no block can span more than two chunks.
int split_cap(int B, int T, int Hkv) {
  const int max_span = (T + kQStep - 1) / kQStep;
  if (max_span <= 2 * kSplitRowSteps) return 0;
  const long long nkt = (T + kColKeys - 1) / kColKeys;
  const long long per_block = (max_span + kSplitRowSteps - 1) / kSplitRowSteps;
  const long long cap = std::min<long long>(2048 / Hkv, (long long)B * nkt * per_block);
  return (int)std::max<long long>(cap, 0);
}
size_t ws_split_bytes(int B, int T, int Hkv, int D) {
  const int capE = split_cap(B, T, Hkv);
  const long long nkt = (T + kColKeys - 1) / kColKeys;
  return round256((size_t)B * nkt * 2 * sizeof(int)) + round256(((size_t)B * nkt + capE) * sizeof(int2)) +
         round256((size_t)capE * Hkv * 2 * kColKeys * D * sizeof(float));
}
static size_t half_delta_bytes(int Hq, int ntok) { return ws_delta_bytes(Hq, ntok) / 2; }

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
  a.flags = p.flags;
  a.scale = p.scale;
  a.scale_log2 = p.scale * 1.4426950408889634f;
  return a;
}

hipError_t launch_kstats(const Problem& p, int BN, int2* kstats) {
  dim3 grid(((p.T + BN - 1) / BN + kWave - 1) / kWave, p.B);
  prof_begin("classify", p.stream);
  hipLaunchKernelGGL(kstats_kernel, grid, dim3(kWave), 0, p.stream, p.evict, p.cu, p.T, p.ntok, BN, kstats);
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_fwd(const Problem& p, const int2* kstats) {
  RowArgs a = row_args(p, kstats);
  const long long nblk = (long long)a.nqt * p.B * p.Hkv * p.nhg;
  dim3 grid((unsigned)nblk), block(64 * p.HG * p.TC);   // 4 waves
  prof_begin("fwd", p.stream);
  if (p.D == 128) hipLaunchKernelGGL(fwd_kernel<128>, grid, block, 0, p.stream, a);
  else hipLaunchKernelGGL(fwd_kernel<64>, grid, block, 0, p.stream, a);
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_bwd_pre(const Problem& p, float* delta) {
  const long long rows = (long long)p.ntok * p.Hq;
  float* lse2 = (float*)((char*)delta + half_delta_bytes(p.Hq, p.ntok));
  dim3 grid((unsigned)((rows + 15) / 16)), block(256);
  prof_begin("bwd_pre", p.stream);
  if (p.D == 128)
    hipLaunchKernelGGL(bwd_pre_kernel<128>, grid, block, 0, p.stream, (const uint16_t*)p.o_in,
                       (const uint16_t*)p.dout, p.lse_in, delta, lse2, p.ntok, p.Hq, p.T, (int)(p.cu != nullptr));
  else
    hipLaunchKernelGGL(bwd_pre_kernel<64>, grid, block, 0, p.stream, (const uint16_t*)p.o_in,
                       (const uint16_t*)p.dout, p.lse_in, delta, lse2, p.ntok, p.Hq, p.T, (int)(p.cu != nullptr));
  prof_end(p.stream);
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const Problem& p, const int2* kstats, const float* delta, void* split_ws) {
  ColArgs a{};
  a.q = (const uint16_t*)p.q;
  a.k = (const uint16_t*)p.k;
  a.v = (const uint16_t*)p.v;
  a.dout = (const uint16_t*)p.dout;
  a.lse = (const float*)((const char*)delta + half_delta_bytes(p.Hq, p.ntok));   // LSE * log2(e)
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
  a.flags = p.flags;
  a.scale = p.scale;
  a.scale_log2 = p.scale * 1.4426950408889634f;
  a.capE = split_cap(p.B, p.T, p.Hkv);
  {
    char* w = (char*)split_ws;
    int* plan = (int*)w;
    w += round256((size_t)p.B * a.nkt * 2 * sizeof(int));
    int2* items = (int2*)w;
    w += round256(((size_t)p.B * a.nkt + a.capE) * sizeof(int2));
    a.plan = plan;
    a.items = items;
    a.part = (float*)w;
    hipLaunchKernelGGL(split_plan_kernel, dim3(1), dim3(1024), 0, p.stream, kstats, p.cu, p.B, p.T, p.ntok, a.nkt,
                       a.capE, plan, items);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const long long nblk = ((long long)a.nkt * p.B + a.capE) * p.Hkv;
  prof_begin("bwd_dkdv", p.stream);
  if (p.D == 128) hipLaunchKernelGGL(dkdv_kernel<128>, dim3((unsigned)nblk), dim3(512), 0, p.stream, a);
  else hipLaunchKernelGGL(dkdv_kernel<64>, dim3((unsigned)nblk), dim3(512), 0, p.stream, a);
  prof_end(p.stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.capE == 0) return e;
  const dim3 rgrid((unsigned)((long long)p.B * a.nkt * p.Hkv * kReduceSplit));
  if (p.D == 128)
    hipLaunchKernelGGL(split_reduce_kernel<128>, rgrid, dim3(256), 0, p.stream, a.plan, a.part, p.cu,
                       (uint16_t*)p.dk, (uint16_t*)p.dv, p.B, p.T, p.ntok, a.nkt, p.Hkv, p.scale);
  else
    hipLaunchKernelGGL(split_reduce_kernel<64>, rgrid, dim3(256), 0, p.stream, a.plan, a.part, p.cu,
                       (uint16_t*)p.dk, (uint16_t*)p.dv, p.B, p.T, p.ntok, a.nkt, p.Hkv, p.scale);
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const Problem& p, const int2* kstats, const float* delta) {
  RowArgs a = row_args(p, kstats);
  a.delta = delta;
  a.lse_in = (const float*)((const char*)delta + half_delta_bytes(p.Hq, p.ntok));   // LSE * log2(e)
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
