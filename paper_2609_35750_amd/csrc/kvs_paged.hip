// gfx950 kernels of the streamed paged KV cache (the inference side of
// KV-streams: Section 2, "KV-streams"; Section 4, "Inference engine
// implementation").  The engine appends one (K, V) entry per generated token
// to a paged cache and drops evicted entries for good; a query attends over
// exactly the entries that are live when it is generated.
//
// Cache layout: K, V [num_blocks][Hkv][block_size][D] bf16 (a block holds one
// contiguous run of block_size rows per KV head); slot_pos [num_blocks *
// block_size] int32 holds the trace position of the token in a slot (slot =
// block * block_size + row), or -1 (empty or evicted).  A sequence's blocks are
// listed in its row of the block table.
//
// Decode: one wave per (sequence, KV head, split).  The wave walks its split's
// cache slots in tiles of 32, gathering each tile's K and V rows from their
// blocks into LDS with asynchronous global-to-LDS copies (double-buffered, no
// workgroup barrier: each wave owns its buffers), computes S^T = K Q^T with the
// G q-heads of the group as the MFMA N columns, masks slots that are empty,
// evicted or past the sequence's last slot, runs the online softmax per
// column and accumulates O^T += V^T P^T.  Partial (max, sum, O) of every split
// go to the workspace; a combine kernel merges them into O and LSE.
#include "kvs_device.h"
#include "kvs_launch.h"

#include <algorithm>

namespace kvs {

// ---------------------------------------------------------------- append / evict
// Token t of the batch goes to cache slot slots[t]; slots outside [0, num_slots) are skipped.
template <int D>
__global__ void __launch_bounds__(256) paged_append_kernel(const uint16_t* __restrict__ kn,
                                                           const uint16_t* __restrict__ vn,
                                                           const int* __restrict__ pos, const int* __restrict__ slots,
                                                           int n, uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                           int* __restrict__ slot_pos, int num_slots, int Hkv, int BS) {
  const long long per_tok = (long long)Hkv * (D / 8);   // 16-byte chunks per token and tensor
  const long long chunks = (long long)n * per_tok;
  for (long long c = (long long)blockIdx.x * blockDim.x + threadIdx.x; c < chunks;
       c += (long long)gridDim.x * blockDim.x) {
    const long long t = c / per_tok, r = c - t * per_tok;
    const int slot = slots[t];
    if ((unsigned)slot >= (unsigned)num_slots) continue;
    const int h = (int)(r / (D / 8)), d8 = (int)(r - (long long)h * (D / 8));
    const long long dst = ((((long long)(slot / BS) * Hkv + h) * BS + slot % BS) * D) + 8 * d8;
    *reinterpret_cast<uint4*>(kc + dst) = *reinterpret_cast<const uint4*>(kn + c * 8);
    *reinterpret_cast<uint4*>(vc + dst) = *reinterpret_cast<const uint4*>(vn + c * 8);
    if (r == 0) slot_pos[slot] = pos[t];
  }
}

__global__ void __launch_bounds__(256) paged_evict_kernel(const int* __restrict__ slots, int n,
                                                          int* __restrict__ slot_pos, int num_slots) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const int slot = slots[i];
    if ((unsigned)slot < (unsigned)num_slots) slot_pos[slot] = -1;
  }
}

// ---------------------------------------------------------------- decode
struct DecodeArgs {
  const uint16_t* q;      // [S][Hq][D]
  const uint16_t* kc;     // [num_blocks][BS][Hkv][D]
  const uint16_t* vc;
  const int* slot_pos;    // [num_blocks * BS]
  const int* table;       // [S][max_blocks]
  const int* nblk;        // [S]
  float* part;            // [S][Hq][nsplit][D]: unnormalised O of each split (relative to its max)
  float* part_ml;         // [S][Hq][nsplit][2]: max (log2 units), sum
  int S, Hq, Hkv, G, max_blocks, BS, num_blocks, nsplit;
  float scale_log2;       // softmax_scale * log2(e)
};

constexpr int kDecTile = 32;   // cache slots per tile

// The 32-slot tile's K or V rows (D = 128: 18 x 16-byte slots per padded LDS
// row, 9 pieces of 64 lanes; D = 64: 9 per row, 4.5 pieces -> 5 with a guard).
template <int D>
struct GatherStager {
  using LY = Lay<D, true>;
  static constexpr int SLOTS = kDecTile * LY::CPRP;
  static constexpr int NI = (SLOTS + kWave - 1) / kWave;
  int row[NI];   // tile row of this lane's 16-byte slot (-1: none)
  int col[NI];   // element column in the source row
  __device__ __forceinline__ void init(int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * kWave + lane;
      const int r = q / LY::CPRP, pc = q - r * LY::CPRP;
      row[i] = q < SLOTS ? r : -1;
      col[i] = (q < SLOTS && pc < LY::CPR) ? 8 * (pc ^ LY::flip(r)) : 0;
    }
  }
  // K and V rows of one tile.  roff: element offset of tile row (lane % 32)
  // in the caches (lanes 0..31, a valid row).  The offsets of all pieces are
  // exchanged first (one LDS round trip), then the copies are issued back to back.
  __device__ __forceinline__ void issue(uint32_t ldsK, uint32_t ldsV, const uint16_t* __restrict__ kb,
                                        const uint16_t* __restrict__ vb, long long roff) const {
    int lo[NI], hi[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = row[i] < 0 ? 0 : row[i];
      lo[i] = __shfl((int)(uint32_t)roff, r);
      hi[i] = __shfl((int)(roff >> 32), r);
    }
    __builtin_amdgcn_sched_barrier(0);   // all exchanges before the first copy
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      if (i * kWave + kWave <= SLOTS || row[i] >= 0) {
        const long long off = (long long)(((uint64_t)(uint32_t)hi[i] << 32) | (uint32_t)lo[i]) + col[i];
        dma_b128_global(kb + off, ldsK + i * kWave * 16);
        dma_b128_global(vb + off, ldsV + i * kWave * 16);
      }
    }
  }
};

// Copies in flight per wave: a ring of kDecRing tiles (K, V and the tile's
// slot_pos values), one ahead of the one being computed.  D = 128 uses 37 KB
// of LDS per wave, so four waves (one per SIMD) share a CU; D = 64 18 KB
// (eight).  A deeper ring costs SIMDs: four stages at two waves per CU
// measured 20% slower on the 64-rollout decode.
constexpr int kDecRing = 2;

// Wait until at most N vector memory operations of this wave are outstanding (N <= 63).
template <int N>
__device__ __forceinline__ void wait_vm_le() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// Every global read of the decode loop is an asynchronous copy to LDS, so all
// of them complete in issue order under one counter and each wait is exact
// (R = kDecRing):
// step n reads the block-table entries of tile n + R - 1 (copied during step
// n - 1), issues the table copy of tile n + R, the K/V copy of tile n + R - 1
// and the copy of its slot_pos values, and computes tile n once at most the
// copies of the R - 1 later steps are outstanding.  (A compiler-visible load
// consumed while copies are in flight would make the compiler wait for all
// of them, since it cannot see them.)
template <int D>
__global__ void __launch_bounds__(64) paged_decode_kernel(DecodeArgs a) {
  constexpr int KS = D / 16, DB = D / 32, PITCH = Lay<D, true>::PITCH, TILE = kDecTile * PITCH, R = kDecRing;
  constexpr int OPS_KV = 2 * GatherStager<D>::NI;   // K and V copy instructions per tile
  constexpr int OPS_STEP = OPS_KV + 2;             // plus the table and slot_pos copies
  static_assert((R - 1) * OPS_STEP < 64, "outstanding copies must fit vmcnt");
  __shared__ __attribute__((aligned(1024))) uint16_t sK[R * TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[R * TILE];
  __shared__ __attribute__((aligned(256))) int sTab[2][kWave];   // block-table entries of a tile's rows
  __shared__ __attribute__((aligned(256))) int sPos[R][kWave];   // slot_pos of a tile's rows

  int wg = blockIdx.x;
  const int sp = wg % a.nsplit;
  wg /= a.nsplit;
  const int g = wg % a.Hkv;
  const int s = wg / a.Hkv;
  const int lane = threadIdx.x, half = lane >> 5, col = lane & 31;
  const auto rl = Lay<D, true>::row_lane(lane);
  const int tl = Lay<D, true>::tr_lo(lane), th = Lay<D, true>::tr_hi(lane);

  // blocks in use by sequence s (clamped to the table width; some slots may be evicted)
  const int nslots = min(max(a.nblk[s], 0), a.max_blocks) * a.BS;
  // the sequence's slots in nsplit equal ranges of whole tiles
  const int per = ((nslots + a.nsplit - 1) / a.nsplit + kDecTile - 1) / kDecTile * kDecTile;
  const int c_begin = min(sp * per, nslots);
  const int c_end = min(c_begin + per, nslots);
  const int ntile = c_end > c_begin ? (c_end - c_begin + kDecTile - 1) / kDecTile : 0;

  // Q^T operand: column n = q-head g * G + n of the group (zero for n >= G)
  const int hcol = g * a.G + col;
  const bool col_ok = col < a.G;
  bf16x8 qreg[KS];
  {
    const uint16_t* qrow = a.q + ((size_t)s * a.Hq + (col_ok ? hcol : g * a.G)) * D + 8 * half;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 u = *reinterpret_cast<const uint4*>(qrow + 16 * ks);
      qreg[ks] = as_bf16x8(col_ok ? u : make_uint4(0u, 0u, 0u, 0u));
    }
  }
  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) acc[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  const int* trow = a.table + (size_t)s * a.max_blocks;
  const long long blk_stride = (long long)a.Hkv * a.BS * D;   // elements per cache block
  const uint16_t* kbase = a.kc + (long long)g * a.BS * D;
  const uint16_t* vbase = a.vc + (long long)g * a.BS * D;
  GatherStager<D> gst;
  gst.init(lane);

  // sequence-local slot index of tile row `col` of tile t (rows past c_end
  // repeat the split's last slot and are masked)
  auto slot_index = [&](int t) __attribute__((always_inline)) { return min(c_begin + t * kDecTile + col, c_end - 1); };
  // copy the block-table entries of tile t's rows (lanes 0..31) into sTab[t & 1]
  auto copy_table = [&](int t) __attribute__((always_inline)) {
    const int c = slot_index(t);
    if (lane < 32) dma_b32_global(trow + c / a.BS, lds_addr(&sTab[t & 1][0]));
  };

  unsigned valid_q[R] = {};   // rows of tiles n .. n + R - 1 that hold a slot of the split (index 0 = tile n)
  if (ntile > 0) copy_table(0);
  wait_vm_le<0>();   // Q and the first table entries are in (no compiler-visible load stays pending in the loop)
  for (int n = -(R - 1); n < ntile; ++n) {
    const int tn = n + R - 1;   // tile whose copies this step issues
    if (tn < ntile) {
      if (n > -(R - 1)) wait_vm_le<OPS_KV + 1>();   // table entries of tile tn have landed
      const int c = slot_index(tn);
      const int blk = sTab[tn & 1][col];
      // a table entry outside the cache reads slot 0 and is masked
      const bool bok = (unsigned)blk < (unsigned)a.num_blocks;
      const int slot = bok ? blk * a.BS + c % a.BS : 0;
      const long long roff = bok ? (long long)blk * blk_stride + (long long)(c % a.BS) * D : 0;
      copy_table(min(tn + 1, ntile - 1));   // always one copy, so that every step issues the same count
      gst.issue(lds_addr(sK + (tn % R) * TILE), lds_addr(sV + (tn % R) * TILE), kbase, vbase, roff);
      if (lane < 32) dma_b32_global(a.slot_pos + slot, lds_addr(&sPos[tn % R][0]));
      valid_q[R - 1] = (unsigned)__ballot(lane < 32 && c_begin + tn * kDecTile + col < c_end && bok);
      if (n >= 0) wait_vm_le<(R - 1) * OPS_STEP>();   // tile n has landed
    } else if (n >= 0) {
      wait_vm_le<0>();
    }
    if (n >= 0) {
      const unsigned live_cur = valid_q[0] & (unsigned)__ballot(lane < 32 && sPos[n % R][col] >= 0);
      const uint16_t* cK = sK + (n % R) * TILE;
      const uint16_t* cV = sV + (n % R) * TILE;
      if (live_cur != 0u) {
        // S^T block: keys on M (tile rows), q-heads on N
        f32x16 sc = f32x16{};
        bf16x8 ka[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) ka[ks] = lds_read_b128(cK + Lay<D, true>::row_at(rl, ks));
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sc = mfma32(ka[ks], qreg[ks], sc);
        // element r <-> tile row 8 (r / 4) + 4 half + r % 4
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 8 * (r >> 2) + 4 * half + (r & 3);
          if (!((live_cur >> row) & 1u)) sc[r] = -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[r]);
        mx = halves_max(mx) * a.scale_log2;
        if (mx > m_run) {   // per column (lane)
          const float alpha = __builtin_amdgcn_exp2f(m_run - mx);   // 0 on the first live tile
          l_run *= alpha;
#pragma unroll
          for (int d = 0; d < DB; ++d)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[d][r] *= alpha;
          m_run = mx;
        }
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sc[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[r], a.scale_log2, -m_use));
          l_run += sc[r];
        }
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          const bf16x8 pb = pack8(sc, 8 * t2);
#pragma unroll
          for (int d = 0; d < DB; ++d) acc[d] = mfma32(tr_operand<D, true>(cV, 16 * t2, 32 * d, tl, th), pb, acc[d]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < R - 1; ++i) valid_q[i] = valid_q[i + 1];
    valid_q[R - 1] = 0u;
  }

  // partial of this split for q-head column `col`
  const float l_tot = halves_sum(l_run);
  if (col_ok) {
    const size_t pidx = ((size_t)s * a.Hq + hcol) * a.nsplit + sp;
    float* dst = a.part + pidx * D;
    if (l_tot > 0.f) {   // an empty split leaves its O unwritten (the merge skips it)
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          *reinterpret_cast<float4*>(dst + 32 * d + 8 * q4 + 4 * half) =
              make_float4(acc[d][4 * q4], acc[d][4 * q4 + 1], acc[d][4 * q4 + 2], acc[d][4 * q4 + 3]);
    }
    if (half == 0) {
      a.part_ml[2 * pidx] = m_run;
      a.part_ml[2 * pidx + 1] = l_tot;
    }
  }
}

// Merge the splits of one (sequence, q-head): one wave, D / 64 values per lane.
template <int D>
__global__ void __launch_bounds__(256) paged_combine_kernel(const float* __restrict__ part,
                                                            const float* __restrict__ part_ml, int rows, int nsplit,
                                                            uint16_t* __restrict__ o, float* __restrict__ lse) {
  const int r = blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float* ml = part_ml + (size_t)r * nsplit * 2;
  float M = -INFINITY;
  for (int i = 0; i < nsplit; ++i) M = fmaxf(M, ml[2 * i]);
  float L = 0.f;
  constexpr int PER = D / 64;
  float x[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) x[e] = 0.f;
  for (int i = 0; i < nsplit; ++i) {
    const float l = ml[2 * i + 1];
    if (l <= 0.f) continue;   // empty split
    const float w = __builtin_amdgcn_exp2f(ml[2 * i] - M);
    L += l * w;
    const float* pv = part + ((size_t)r * nsplit + i) * D + PER * lane;
#pragma unroll
    for (int e = 0; e < PER; ++e) x[e] += pv[e] * w;
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  uint16_t* orow = o + (size_t)r * D + PER * lane;
#pragma unroll
  for (int e = 0; e < PER; ++e) orow[e] = __builtin_bit_cast(uint16_t, (__bf16)(x[e] * inv));
  if (lane == 0) lse[r] = L > 0.f ? (M + __log2f(L)) * 0.6931471805599453f : -INFINITY;
}

template __global__ void paged_append_kernel<64>(const uint16_t*, const uint16_t*, const int*, const int*, int,
                                                 uint16_t*, uint16_t*, int*, int, int, int);
template __global__ void paged_append_kernel<128>(const uint16_t*, const uint16_t*, const int*, const int*, int,
                                                  uint16_t*, uint16_t*, int*, int, int, int);
template __global__ void paged_decode_kernel<64>(DecodeArgs);
template __global__ void paged_decode_kernel<128>(DecodeArgs);
template __global__ void paged_combine_kernel<64>(const float*, const float*, int, int, uint16_t*, float*);
template __global__ void paged_combine_kernel<128>(const float*, const float*, int, int, uint16_t*, float*);

// ---------------------------------------------------------------- launchers
// Key splits per (sequence, KV head): enough waves for one round of the
// resident ones (D = 128: four per CU, D = 64: eight; each sequence's live
// slots are cut into that many equal ranges on the device), at most one split
// per four tiles of the table width.
int paged_nsplit(int S, int Hkv, int max_blocks, int BS, int D) {
  const long long max_slots = (long long)max_blocks * BS;
  const long long units = (long long)S * Hkv;
  long long splits = ((D == 128 ? 4ll : 8ll) * 256 + units - 1) / units;
  splits = std::min(splits, std::max(1ll, max_slots / (4 * kDecTile)));
  return (int)std::max(1ll, splits);
}
size_t paged_ws_bytes(int S, int Hq, int D, int nsplit) {
  const size_t rows = (size_t)S * Hq * nsplit;
  return ((rows * D * sizeof(float) + 255) & ~(size_t)255) + ((rows * 2 * sizeof(float) + 255) & ~(size_t)255);
}

hipError_t launch_paged_append(const void* kn, const void* vn, const int* pos, const int* slots, int n, void* kc,
                               void* vc, int* slot_pos, int num_slots, int BS, int Hkv, int D, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const long long chunks = (long long)n * Hkv * (D / 8);
  const int blocks = (int)std::min<long long>((chunks + 255) / 256, 65535);
  if (D == 128)
    hipLaunchKernelGGL(paged_append_kernel<128>, dim3(blocks), dim3(256), 0, stream, (const uint16_t*)kn,
                       (const uint16_t*)vn, pos, slots, n, (uint16_t*)kc, (uint16_t*)vc, slot_pos, num_slots, Hkv, BS);
  else
    hipLaunchKernelGGL(paged_append_kernel<64>, dim3(blocks), dim3(256), 0, stream, (const uint16_t*)kn,
                       (const uint16_t*)vn, pos, slots, n, (uint16_t*)kc, (uint16_t*)vc, slot_pos, num_slots, Hkv, BS);
  return hipGetLastError();
}

hipError_t launch_paged_evict(const int* slots, int n, int* slot_pos, int num_slots, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int blocks = std::min((n + 255) / 256, 4096);
  hipLaunchKernelGGL(paged_evict_kernel, dim3(blocks), dim3(256), 0, stream, slots, n, slot_pos, num_slots);
  return hipGetLastError();
}

hipError_t launch_paged_decode(const PagedDecode& p) {
  DecodeArgs a{};
  a.q = (const uint16_t*)p.q;
  a.kc = (const uint16_t*)p.k_cache;
  a.vc = (const uint16_t*)p.v_cache;
  a.slot_pos = p.slot_pos;
  a.table = p.block_table;
  a.nblk = p.seq_blocks;
  a.S = p.S;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.G = p.Hq / p.Hkv;
  a.max_blocks = p.max_blocks;
  a.BS = p.block_size;
  a.num_blocks = p.num_blocks;
  a.nsplit = paged_nsplit(p.S, p.Hkv, p.max_blocks, p.block_size, p.D);
  a.part = (float*)p.ws;
  const size_t rows = (size_t)p.S * p.Hq * a.nsplit;
  a.part_ml = (float*)((char*)p.ws + ((rows * p.D * sizeof(float) + 255) & ~(size_t)255));
  a.scale_log2 = p.scale * 1.4426950408889634f;
  const dim3 grid((unsigned)((long long)p.S * p.Hkv * a.nsplit));
  prof_begin("paged_decode", p.stream);
  if (p.D == 128) hipLaunchKernelGGL(paged_decode_kernel<128>, grid, dim3(64), 0, p.stream, a);
  else hipLaunchKernelGGL(paged_decode_kernel<64>, grid, dim3(64), 0, p.stream, a);
  prof_end(p.stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rows_out = p.S * p.Hq;
  const dim3 cgrid((unsigned)((rows_out + 3) / 4));
  if (p.D == 128)
    hipLaunchKernelGGL(paged_combine_kernel<128>, cgrid, dim3(256), 0, p.stream, a.part, a.part_ml, rows_out,
                       a.nsplit, (uint16_t*)p.o, p.lse);
  else
    hipLaunchKernelGGL(paged_combine_kernel<64>, cgrid, dim3(256), 0, p.stream, a.part, a.part_ml, rows_out,
                       a.nsplit, (uint16_t*)p.o, p.lse);
  return hipGetLastError();
}

}  // namespace kvs
