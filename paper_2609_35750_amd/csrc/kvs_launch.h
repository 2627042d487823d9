// Internal interface between the C ABI layer (kvs_api.cpp) and the kernel
// launchers (kvs_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace kvs {

// Problem description after host-side validation.
struct Problem {
  const void* q;
  const void* k;
  const void* v;
  const void* o_in;      // backward: forward output O
  const void* dout;      // backward: dO
  const float* lse_in;   // backward: forward LSE
  const int32_t* evict;
  const int32_t* cu;     // NULL: fixed length
  void* o;               // forward output
  float* lse;            // forward output
  void* dq;
  void* dk;
  void* dv;
  int B;
  int T;        // fixed: trace length; varlen: max_seqlen
  int ntok;     // total packed tokens
  int Hq, Hkv, D, G;
  int HG, TC, nhg;   // q-heads per workgroup, 32-token chunks per workgroup, head groups per KV head
  int flags;         // tile-classifier switches (kFlagNoEmptySkip, kFlagFullAsPartial); 0 normally
  float scale;
  void* ws;
  hipStream_t stream;
};

// Workspace pieces (byte offsets from the workspace start).
size_t ws_kstats_bytes(int B, int ntok);

// Library-owned scratch of the allocation-free forward: kNoAllocScratchBytes
// per GPU (device address of this device's copy in *ptr; taken once per device).
constexpr size_t kNoAllocScratchBytes = 256 * 1024;
constexpr int kMaxDevices = 64;
hipError_t noalloc_scratch(void** ptr);
size_t ws_delta_bytes(int Hq, int ntok);
size_t ws_split_bytes(int B, int T, int Hkv, int D);

// Launchers.  Each returns the hipError_t of its launch(es).
hipError_t launch_kstats(const Problem& p, int BN, int2* kstats);
hipError_t launch_fwd(const Problem& p, const int2* kstats);
hipError_t launch_bwd_pre(const Problem& p, float* delta);
hipError_t launch_bwd_dkdv(const Problem& p, const int2* kstats, const float* delta, void* split_ws);
hipError_t launch_bwd_dq(const Problem& p, const int2* kstats, const float* delta);
hipError_t launch_classify(const int32_t* evict, const int32_t* cu, int B, int T, int BM, int BN,
                           uint8_t* out, hipStream_t stream);
hipError_t launch_check(const int32_t* evict, const int32_t* cu, int B, int T, int ntok,
                        int64_t* first_bad, int* cu_bad, hipStream_t stream);

// Paged decode over the streamed KV cache (after host-side validation).
struct PagedDecode {
  const void* q;            // [S][Hq][D] bf16
  const void* k_cache;      // [num_blocks][Hkv][block_size][D] bf16
  const void* v_cache;
  const int32_t* slot_pos;  // [num_blocks * block_size]
  const int32_t* block_table;   // [S][max_blocks]
  const int32_t* seq_blocks;    // [S]
  void* o;                  // [S][Hq][D] bf16
  float* lse;               // [S][Hq]
  int S, Hq, Hkv, D, max_blocks, block_size, num_blocks;
  float scale;
  void* ws;
  hipStream_t stream;
};
int paged_nsplit(int S, int Hkv, int max_blocks, int BS, int D);
size_t paged_ws_bytes(int S, int Hq, int D, int nsplit);
hipError_t launch_paged_append(const void* kn, const void* vn, const int* pos, const int* slots, int n, void* kc,
                               void* vc, int* slot_pos, int num_slots, int BS, int Hkv, int D, hipStream_t stream);
hipError_t launch_paged_evict(const int* slots, int n, int* slot_pos, int num_slots, hipStream_t stream);
hipError_t launch_paged_decode(const PagedDecode& p);

// Per-kernel event bracketing (benchmark timing).
void prof_begin(const char* name, hipStream_t s);
void prof_end(hipStream_t s);

}  // namespace kvs
