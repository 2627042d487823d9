/*
 * kvs.h -- C ABI of the eviction-masked attention library (libkvs.so) for
 * AMD Instinct MI355X (gfx950).
 *
 * What it computes.  KV-streams (Section 2, paragraph "KV-streams") keeps the
 * retained keys and values of a compacted agent trace at their original
 * positions and reproduces each compaction in the trainer with an attention
 * mask over one continuous trace, in a single forward pass.  The engine
 * drops evicted entries for good (Section 7, second paragraph), so every key
 * token j of a trace carries one eviction index evict_at[j], and query i
 * attends to key j iff
 *
 *        j <= i < evict_at[j]      (evict_at[j] >= L, e.g. INT32_MAX, = never evicted)
 *
 * For q-head h of KV head g = h / (Hq / Hkv) (contiguous GQA groups):
 *        s_ij  = softmax_scale * <Q_i^h, K_j^g>
 *        LSE_i = ln sum_{visible j} exp(s_ij)
 *        O_i   = sum_{visible j} exp(s_ij - LSE_i) V_j^g
 * and the backward gives dQ, dK, dV of sum(dO * O) (dK, dV summed over the
 * q-heads of each group).  Every query sees at least itself (evict_at[j] > j
 * is required), so no row is empty.
 *
 * Conventions shared by every entry point:
 *  - Tensor pointers are DEVICE pointers owned by the caller; the library
 *    never allocates device memory and keeps no per-call state.  Scratch space
 *    comes from the caller's workspace (size from the *_workspace query; any
 *    256-byte aligned device buffer of at least that size).  The only
 *    process-wide state is that of kvs_check_evict_at (calls are serialised)
 *    and of the benchmark timers kvs_prof_* (see there).
 *  - bf16 tensors are row-major with D innermost:
 *       fixed length:  Q, O, dO, dQ [B][T][Hq][D];  K, V, dK, dV [B][T][Hkv][D]
 *       varlen:        Q, O, dO, dQ [Ntot][Hq][D];  K, V, dK, dV [Ntot][Hkv][D]
 *    LSE is fp32, natural log: fixed [B][Hq][T], varlen [Hq][Ntot].
 *    evict_at is int32: fixed [B][T], varlen [Ntot]; values are trace-local
 *    token indices.  Tensor pointers must be 16-byte aligned.
 *  - cu_seqlens (varlen) is a device int32 array [B+1]: cu[0] = 0,
 *    cu[B] = Ntot, non-decreasing; trace b is tokens [cu[b], cu[b+1]).
 *    No attention crosses traces.  max_seqlen must be >= every trace length.
 *    The host cannot see these offsets, so the kernels never trust them for
 *    addressing: each trace start is clamped to [0, Ntot], its end to
 *    [start, Ntot] and its length to max_seqlen.  A malformed cu_seqlens (or a
 *    trace longer than max_seqlen) gives unspecified results but no access
 *    outside the caller's buffers; kvs_check_evict_at reports it.
 *  - `stream` is a hipStream_t (NULL = the null stream).  Calls only enqueue
 *    work on it and return; none synchronizes except kvs_check_evict_at.
 *  - Outputs are overwritten, never accumulated.
 *  - An empty batch (Ntot = 0, e.g. varlen traces that are all empty) is
 *    valid: shapes, softmax_scale and flags are still checked, then the call
 *    returns KVS_OK without looking at any tensor pointer or the workspace
 *    (zero-size buffers may be NULL; the varlen calls still need cu_seqlens)
 *    and without enqueuing work.
 *  - Supported: D in {64, 128}; 1 <= Hkv <= Hq, Hq % Hkv == 0, Hq / Hkv <= 64;
 *    T (max_seqlen) <= 1048576.  Other shapes return KVS_ERR_SHAPE or
 *    KVS_ERR_UNSUPPORTED.
 *  - Arguments are validated on the host before any HIP call, so invalid
 *    calls fail the same way on machines without a GPU.
 *  - Results are unspecified if some evict_at[j] <= j (trace-local); use
 *    kvs_check_evict_at to detect that.
 */
#ifndef KVS_H_
#define KVS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVS_ABI_VERSION 3

typedef enum {
  KVS_OK = 0,
  KVS_ERR_NULL = 1,         /* a required pointer is NULL */
  KVS_ERR_SHAPE = 2,        /* bad sizes: B,T,Hq,Hkv < 1, Hq % Hkv != 0, D not 64/128, bad BM/BN */
  KVS_ERR_ALIGN = 3,        /* a tensor pointer is not 16-byte aligned (workspace: 256-byte) */
  KVS_ERR_WORKSPACE = 4,    /* workspace smaller than the *_workspace query */
  KVS_ERR_EVICT = 5,        /* invalid evict_at (only kvs_check_evict_at reports it) */
  KVS_ERR_HIP = 6,          /* a HIP launch or runtime call failed; see kvs_last_error() */
  KVS_ERR_UNSUPPORTED = 7,  /* valid but outside the supported limits above */
  KVS_ERR_CAPACITY = 8,     /* paged cache: no free block, or a sequence's block table is full */
  KVS_ERR_STATE = 9         /* paged cache: position already cached, or not cached */
} kvs_status_t;

/* ABI version of the loaded library (KVS_ABI_VERSION it was built with). */
int kvs_abi_version(void);

/* Static English text for a status code; never NULL. */
const char* kvs_status_string(kvs_status_t status);

/* Detail of the most recent failure on the calling thread (which argument,
 * which HIP error); "" if none.  Valid until the next call on that thread. */
const char* kvs_last_error(void);

/* ---------------------------------------------------------------- forward
 * Eviction-masked attention forward (Section 2, "KV-streams": one pass over
 * the continuous trace with a mask that blocks each deleted span).
 * Writes O (bf16) and LSE (fp32, natural log).  B traces of equal length T.
 */
size_t kvs_evict_attn_fwd_workspace(int B, int T, int Hq, int Hkv, int D);
kvs_status_t kvs_evict_attn_fwd(const void* Q, const void* K, const void* V,
                                const int32_t* evict_at,
                                void* O, float* LSE,
                                int B, int T, int Hq, int Hkv, int D, float softmax_scale,
                                void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------- backward
 * Gradients of sum(dO * O) for the forward above: dQ, dK, dV (bf16, shapes
 * of Q, K, V).  O and LSE must be the forward's outputs for the same inputs.
 */
size_t kvs_evict_attn_bwd_workspace(int B, int T, int Hq, int Hkv, int D);
kvs_status_t kvs_evict_attn_bwd(const void* dO, const void* Q, const void* K, const void* V,
                                const void* O, const float* LSE, const int32_t* evict_at,
                                void* dQ, void* dK, void* dV,
                                int B, int T, int Hq, int Hkv, int D, float softmax_scale,
                                void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------- varlen
 * The same computations over B traces packed back to back (several rollouts
 * in one batch, each its own continuous trace; Section 2).  Layouts as above
 * with the varlen shapes; evict_at values are local to each trace.
 */
size_t kvs_evict_attn_varlen_fwd_workspace(int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D);
kvs_status_t kvs_evict_attn_varlen_fwd(const void* Q, const void* K, const void* V,
                                       const int32_t* evict_at, const int32_t* cu_seqlens,
                                       void* O, float* LSE,
                                       int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D,
                                       float softmax_scale,
                                       void* workspace, size_t workspace_bytes, void* stream);
size_t kvs_evict_attn_varlen_bwd_workspace(int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D);
kvs_status_t kvs_evict_attn_varlen_bwd(const void* dO, const void* Q, const void* K, const void* V,
                                       const void* O, const float* LSE,
                                       const int32_t* evict_at, const int32_t* cu_seqlens,
                                       void* dQ, void* dK, void* dV,
                                       int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D,
                                       float softmax_scale,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------- consistency switches
 * The forward and backward skip EMPTY tiles and evaluate no mask on FULL
 * tiles.  These switches turn the shortcuts off without changing anything
 * else (same kernels, same tile order, same row and key ranges), so that a
 * caller can check that the shortcuts are exact: the mask must block the
 * whole deleted span (Section 2, "KV-streams"), so a skipped tile holds no
 * visible entry and a FULL tile no masked one, and every output (O, LSE, dQ,
 * dK, dV) must come out bit-identical with and without them.  They cost
 * time and are meant for tests.
 *   KVS_FLAG_NO_EMPTY_SKIP    process every key tile of the range a row
 *                             block walks (and every row block of the range a
 *                             key block walks), masking the EMPTY ones
 *   KVS_FLAG_FULL_AS_PARTIAL  evaluate the per-element mask on FULL tiles
 *
 * kvs_evict_attn_{fwd,bwd}_ex take either layout: cu_seqlens NULL means B
 * fixed-length traces of max_seqlen tokens (Ntot must be B * max_seqlen; the
 * fixed-length layouts above), otherwise the varlen layouts.  Workspace: the
 * size the matching non-_ex query gives.  Unknown flag bits give
 * KVS_ERR_UNSUPPORTED; flags = 0 is the plain call.
 */
#define KVS_FLAG_NO_EMPTY_SKIP 1u
#define KVS_FLAG_FULL_AS_PARTIAL 2u

kvs_status_t kvs_evict_attn_fwd_ex(const void* Q, const void* K, const void* V,
                                   const int32_t* evict_at, const int32_t* cu_seqlens,
                                   void* O, float* LSE,
                                   int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D,
                                   float softmax_scale, unsigned flags,
                                   void* workspace, size_t workspace_bytes, void* stream);
kvs_status_t kvs_evict_attn_bwd_ex(const void* dO, const void* Q, const void* K, const void* V,
                                   const void* O, const float* LSE,
                                   const int32_t* evict_at, const int32_t* cu_seqlens,
                                   void* dQ, void* dK, void* dV,
                                   int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D,
                                   float softmax_scale, unsigned flags,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------- allocation-free forward
 * For callers that cannot allocate device memory or hand over a workspace:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  kvs_evict_attn_fwd_ex (flags 0) without the workspace: the
 * per-key-tile statistics the forward needs go to a library-owned device
 * array of 256 KiB, one copy per GPU, held from the first call on that GPU
 * until the process ends.  Layouts and cu_seqlens as in the *_ex calls.
 * The call allocates nothing (no hipMalloc, no hipFree, no allocating library
 * routine).  Limit: B + Ntot / 64 + 2 <= 32768 key tiles (one trace of up to
 * the 1,048,576-token maximum, or e.g. 8 traces of 110k tokens); beyond it
 * KVS_ERR_UNSUPPORTED.  Every call on a GPU uses that GPU's one array, which
 * keeps the last call's contents (each entry a kernel reads is written
 * earlier in the same call): calls that overlap on one GPU (several streams
 * or threads) race and give wrong results, so issue them on one stream.
 */
kvs_status_t kvs_evict_attn_fwd_noalloc(const void* Q, const void* K, const void* V,
                                        const int32_t* evict_at, const int32_t* cu_seqlens,
                                        void* O, float* LSE,
                                        int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D,
                                        float softmax_scale, void* stream);

/* ---------------------------------------------------------------- tile classes
 * Class of every BM x BN tile of the mask: 0 = EMPTY (no visible element,
 * skipped), 1 = PARTIAL (per-element mask), 2 = FULL (every element
 * visible).  Tiles start at each trace's first token; elements outside the
 * trace count as masked.  Output: per-trace grids, each row-major
 * [ceil(L_b/BM)][ceil(L_b/BN)], concatenated in trace order into tile_class
 * (device uint8, caller-sized).  cu_seqlens NULL means B traces of length T;
 * otherwise T is Ntot.  The attention kernels classify with the same rule
 * (BM multiple of 16 in [16, 256], BN in {32, 64, 128}).
 */
kvs_status_t kvs_classify_tiles(const int32_t* evict_at, const int32_t* cu_seqlens, int B, int T,
                                int BM, int BN, uint8_t* tile_class, void* stream);

/* Number of bytes kvs_classify_tiles writes when the trace lengths are known
 * on the host (lengths: host int32 [B]). */
size_t kvs_classify_tiles_size(const int32_t* lengths, int B, int BM, int BN);

/* ---------------------------------------------------------------- validation
 * Synchronous check that every key is visible to itself (evict_at[j] > j,
 * trace-local).  On return *first_bad (host) is the packed index of the first
 * offending key, or -1.  Returns KVS_ERR_EVICT if one exists, KVS_ERR_SHAPE if
 * cu_seqlens is not 0 = cu[0] <= ... <= cu[B] = T.  cu_seqlens as in
 * kvs_classify_tiles.  Blocks until the stream reaches it.  The result passes
 * through device globals of the library, one copy per GPU, so calls are
 * serialised within a process (thread-safe; concurrent calls wait).
 */
kvs_status_t kvs_check_evict_at(const int32_t* evict_at, const int32_t* cu_seqlens, int B, int T,
                                int64_t* first_bad, void* stream);

/* ---------------------------------------------------------------- timing
 * Per-kernel timing for benchmarks.  While enabled, each call brackets every
 * kernel it launches with HIP events on the call's stream.  kvs_prof_read
 * waits for the recorded events and returns, for the kernel named `name`
 * ("classify", "fwd", "bwd_pre", "bwd_dkdv", "bwd_dq", "paged_decode"), the
 * number of launches and their total duration in milliseconds.  The records
 * are process-wide (every thread's launches land in one list, guarded by a
 * lock), so enable timing only while the calls to be timed are the only
 * ones running; meant for benchmark drivers.
 */
void kvs_prof_enable(int on);
void kvs_prof_reset(void);
kvs_status_t kvs_prof_read(const char* name, int* launches, double* total_ms);


/* ================================================================ streamed paged KV cache
 * The inference side of KV-streams (Section 2, "KV-streams"; Section 4,
 * "Inference engine implementation"): the engine appends one (K, V) entry per
 * generated token to a paged cache, evicts entries directly in the cache when
 * a compaction fires (they never come back), and each query attends over
 * exactly the entries that are live when it is generated.  Decoding token i
 * of a trace therefore computes row i of the eviction-masked attention above
 * (keys j <= i with evict_at[j] > i), which is what lets the trainer replay a
 * whole rollout in one masked pass.  Block sizes: 16 (the vLLM setup, turns
 * padded to 16 tokens) or 1 (the SGLang setup); any size in [1, 64] works.
 *
 * Device cache (caller-owned, allocated once):
 *   K_cache, V_cache  bf16 [num_blocks][Hkv][block_size][D]  (16-byte aligned; a
 *                     block holds one contiguous run of block_size rows per KV head)
 *   slot_pos          int32 [num_blocks * block_size]: trace position of the
 *                     token held by each slot, -1 for an empty or evicted slot.
 *                     Must be filled with -1 before first use.
 * Host bookkeeping: a block manager (kvs_bm_*) hands out slots, drops
 * evicted entries, frees blocks with no live entry and produces the block
 * tables the decode call reads:
 *   block_table  int32 [num_seqs][max_blocks]: a sequence's blocks in
 *                allocation order (entries past seq_blocks[s] are ignored)
 *   seq_blocks   int32 [num_seqs]
 * A slot of a block stays allocated until the whole block is free, so the
 * decode call masks the evicted slots of partly evicted blocks by slot_pos.
 */

/* ---- host block manager (host memory only; not thread-safe; no HIP calls) */
typedef struct kvs_block_manager kvs_block_manager;

/* New manager of num_blocks cache blocks of block_size slots for num_seqs
 * sequences of at most max_blocks blocks each (*out, host).  KVS_ERR_SHAPE for
 * non-positive sizes or block_size > 64, KVS_ERR_UNSUPPORTED if
 * num_blocks * block_size exceeds INT32_MAX. */
kvs_status_t kvs_bm_create(int num_blocks, int block_size, int num_seqs, int max_blocks,
                           kvs_block_manager** out);
void kvs_bm_destroy(kvs_block_manager* bm);

/* Reserve slots for n tokens of sequence seq at trace positions pos[0..n)
 * (host arrays); slots[i] receives the slot of pos[i].  Tokens fill the tail
 * of the sequence's last block, then fresh blocks.  All-or-nothing:
 * KVS_ERR_CAPACITY (no free block / table full) or KVS_ERR_STATE (a position
 * already cached or repeated) leave the manager unchanged. */
kvs_status_t kvs_bm_append(kvs_block_manager* bm, int seq, const int32_t* pos, int n, int32_t* slots);

/* Evict the entries of sequence seq at trace positions pos[0..n); slots[i]
 * receives the slot that held pos[i] (pass them to kvs_paged_evict).  Blocks
 * left without a live entry return to the free list and leave the sequence's
 * table.  All-or-nothing; KVS_ERR_STATE if a position is not cached or repeated. */
kvs_status_t kvs_bm_evict(kvs_block_manager* bm, int seq, const int32_t* pos, int n, int32_t* slots);

/* Drop sequence seq entirely: writes its live slots (sorted; `slots` must hold
 * kvs_bm_live(bm, seq) entries) and their count, and frees all its blocks. */
kvs_status_t kvs_bm_release(kvs_block_manager* bm, int seq, int32_t* slots, int* n_slots);

/* Host copies of block_table [num_seqs][max_blocks] (unused entries 0) and seq_blocks [num_seqs]. */
kvs_status_t kvs_bm_tables(const kvs_block_manager* bm, int32_t* block_table, int32_t* seq_blocks);

/* Free blocks; live entries of sequence seq (-1 for a bad index or NULL manager). */
int kvs_bm_free_blocks(const kvs_block_manager* bm);
int kvs_bm_live(const kvs_block_manager* bm, int seq);

/* ---- device updates (enqueued on `stream`) */

/* Write n new tokens into the cache: K_new, V_new bf16 [n][Hkv][D] go to
 * slots[0..n) of K_cache, V_cache and slot_pos[slots[t]] = positions[t] (slot = block * block_size + row)
 * (positions, slots: device int32 [n]).  Slots outside [0, num_blocks *
 * block_size) are skipped (the device cannot report them). */
kvs_status_t kvs_paged_append(const void* K_new, const void* V_new, const int32_t* positions,
                              const int32_t* slots, int n, void* K_cache, void* V_cache, int32_t* slot_pos,
                              int num_blocks, int block_size, int Hkv, int D, void* stream);

/* Mark slots[0..n) (device int32) evicted: slot_pos = -1.  Out-of-range slots are skipped. */
kvs_status_t kvs_paged_evict(const int32_t* slots, int n, int32_t* slot_pos, int num_blocks, int block_size,
                             void* stream);

/* ---- decode attention over the live cache
 * One query token per sequence: Q, O bf16 [num_seqs][Hq][D], LSE fp32
 * [num_seqs][Hq] (natural log).  Sequence s attends over every slot of its
 * first seq_blocks[s] table blocks whose slot_pos is >= 0, with q-head h on KV
 * head h / (Hq / Hkv).  A sequence with no live slot gets O = 0, LSE = -inf.
 * Device inputs that the host cannot see are clamped, never trusted for
 * addressing: seq_blocks to [0, max_blocks]; a table entry outside
 * [0, num_blocks) reads nothing and counts as evicted.
 * Supported: D in {64, 128}; Hq / Hkv <= 32; block_size in [1, 64];
 * num_blocks * block_size <= INT32_MAX.  Workspace: fp32 partials of the
 * key splits (size from the query below, 256-byte aligned). */
size_t kvs_paged_decode_workspace(int num_seqs, int Hq, int Hkv, int D, int max_blocks, int block_size);
kvs_status_t kvs_paged_decode(const void* Q, const void* K_cache, const void* V_cache, const int32_t* slot_pos,
                              const int32_t* block_table, const int32_t* seq_blocks, void* O, float* LSE,
                              int num_seqs, int Hq, int Hkv, int D, int num_blocks, int block_size,
                              int max_blocks, float softmax_scale, void* workspace, size_t workspace_bytes,
                              void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVS_H_ */
