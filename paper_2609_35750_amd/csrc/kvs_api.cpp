// C ABI of libkvs: argument validation, workspace layout and launch order.
// Validation runs before any HIP call, so invalid calls fail identically on
// machines without a GPU.
#include "kvs.h"

#include <hip/hip_runtime_api.h>

#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kvs_cache.h"
#include "kvs_launch.h"

namespace {

thread_local std::string t_err;

kvs_status_t fail(kvs_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  t_err = buf;
  return st;
}

kvs_status_t hip_fail(hipError_t e, const char* where) {
  return fail(KVS_ERR_HIP, "%s: %s (%d)", where, hipGetErrorString(e), (int)e);
}

constexpr int kMaxSeq = 1 << 20;
constexpr int kMaxGroup = 64;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Shape rules shared by every attention entry point.
kvs_status_t check_dims(int B, int T, long long ntok, int Hq, int Hkv, int D) {
  if (B < 1 || T < 1 || Hq < 1 || Hkv < 1)
    return fail(KVS_ERR_SHAPE, "B, T (max_seqlen), Hq, Hkv must be >= 1 (got %d, %d, %d, %d)", B, T, Hq, Hkv);
  if (Hq % Hkv != 0) return fail(KVS_ERR_SHAPE, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
  if (D != 64 && D != 128) return fail(KVS_ERR_SHAPE, "head dim D must be 64 or 128 (got %d)", D);
  if (ntok < 0) return fail(KVS_ERR_SHAPE, "Ntot must be >= 0");
  if (T > kMaxSeq) return fail(KVS_ERR_UNSUPPORTED, "sequence length %d above the supported %d", T, kMaxSeq);
  if (Hq / Hkv > kMaxGroup) return fail(KVS_ERR_UNSUPPORTED, "GQA group size %d above %d", Hq / Hkv, kMaxGroup);
  if (ntok * (long long)Hq * D >= (1ll << 40))
    return fail(KVS_ERR_UNSUPPORTED, "tensor of %lld elements too large", ntok * (long long)Hq * D);
  if (ntok > 0x7fffffffll) return fail(KVS_ERR_UNSUPPORTED, "Ntot above INT32_MAX");
  return KVS_OK;
}

// Workgroup shape of the row kernels: 4 waves, HG q-heads of one GQA group
// (4, 2 or 1, whichever divides G) times TC = 4 / HG chunks of 32 tokens, so
// each K/V tile staged in LDS serves 128 (row, q-head) pairs and two
// workgroups share a CU whatever the group size.
void head_grouping(kvs::Problem& p) {
  const int hg = p.G % 4 == 0 ? 4 : (p.G % 2 == 0 ? 2 : 1);
  p.HG = hg;
  p.TC = 4 / hg;
  p.nhg = p.G / hg;
}

size_t fwd_ws(int B, long long ntok) { return kvs::ws_kstats_bytes(B, (int)ntok); }
size_t bwd_ws(int B, int T, long long ntok, int Hq, int Hkv, int D) {
  return kvs::ws_kstats_bytes(B, (int)ntok) + kvs::ws_delta_bytes(Hq, (int)ntok) + kvs::ws_split_bytes(B, T, Hkv, D);
}

kvs_status_t check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return KVS_OK;
  if (!ws) return fail(KVS_ERR_NULL, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & 255u) != 0) return fail(KVS_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (have < need) return fail(KVS_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", have, need);
  return KVS_OK;
}

#define REQUIRE_PTR(p, name)                                         \
  do {                                                               \
    if (!(p)) return fail(KVS_ERR_NULL, "%s is NULL", name);         \
    if (!aligned16(p)) return fail(KVS_ERR_ALIGN, "%s not 16-byte aligned", name); \
  } while (0)

kvs_status_t run_fwd(kvs::Problem& p) {
  head_grouping(p);
  int2* kstats = (int2*)p.ws;
  hipError_t e = kvs::launch_kstats(p, 64, kstats);
  if (e != hipSuccess) return hip_fail(e, "key-tile statistics launch");
  e = kvs::launch_fwd(p, kstats);
  if (e != hipSuccess) return hip_fail(e, "forward launch");
  return KVS_OK;
}

kvs_status_t run_bwd(kvs::Problem& p) {
  head_grouping(p);
  int2* kstats = (int2*)p.ws;
  float* delta = (float*)((char*)p.ws + kvs::ws_kstats_bytes(p.B, p.ntok));
  hipError_t e = kvs::launch_kstats(p, 64, kstats);
  if (e != hipSuccess) return hip_fail(e, "key-tile statistics launch");
  e = kvs::launch_bwd_pre(p, delta);
  if (e != hipSuccess) return hip_fail(e, "backward preprocess launch");
  void* split_ws = (char*)delta + kvs::ws_delta_bytes(p.Hq, p.ntok);
  e = kvs::launch_bwd_dkdv(p, kstats, delta, split_ws);
  if (e != hipSuccess) return hip_fail(e, "dK/dV launch");
  e = kvs::launch_bwd_dq(p, kstats, delta);
  if (e != hipSuccess) return hip_fail(e, "dQ launch");
  return KVS_OK;
}

// ---------------------------------------------------------------- timing records
// Process-wide and only for benchmark drivers: the records are shared (under
// g_prof_mu), the open bracket of a launch is per thread.
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
std::atomic<bool> g_prof{false};
std::mutex g_prof_mu;
std::vector<ProfRec> g_recs;
thread_local const char* t_pending = nullptr;
thread_local hipEvent_t t_pending_ev = nullptr;

// kvs_check_evict_at keeps its result in device globals of the library; calls
// are serialised (each one synchronises its stream before it returns).
std::mutex g_check_mu;

}  // namespace

namespace kvs {
void prof_begin(const char* name, hipStream_t s) {
  if (!g_prof.load()) return;
  hipEvent_t ev;
  if (hipEventCreate(&ev) != hipSuccess) return;
  (void)hipEventRecord(ev, s);
  t_pending = name;
  t_pending_ev = ev;
}
void prof_end(hipStream_t s) {
  if (!g_prof.load() || !t_pending_ev) return;
  hipEvent_t ev;
  if (hipEventCreate(&ev) != hipSuccess) return;
  (void)hipEventRecord(ev, s);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_recs.push_back({t_pending, t_pending_ev, ev});
  t_pending_ev = nullptr;
}
}  // namespace kvs

extern "C" {

int kvs_abi_version(void) { return KVS_ABI_VERSION; }

const char* kvs_status_string(kvs_status_t s) {
  switch (s) {
    case KVS_OK: return "ok";
    case KVS_ERR_NULL: return "null pointer";
    case KVS_ERR_SHAPE: return "invalid shape";
    case KVS_ERR_ALIGN: return "misaligned pointer";
    case KVS_ERR_WORKSPACE: return "workspace too small";
    case KVS_ERR_EVICT: return "invalid evict_at (some evict_at[j] <= j)";
    case KVS_ERR_HIP: return "HIP runtime error";
    case KVS_ERR_UNSUPPORTED: return "unsupported configuration";
    case KVS_ERR_CAPACITY: return "paged cache capacity exceeded";
    case KVS_ERR_STATE: return "paged cache state conflict";
  }
  return "unknown status";
}

const char* kvs_last_error(void) { return t_err.c_str(); }

size_t kvs_evict_attn_fwd_workspace(int B, int T, int Hq, int Hkv, int D) {
  if (B < 1 || T < 1) return 0;
  (void)Hq; (void)Hkv; (void)D;
  return fwd_ws(B, (long long)B * T);
}

size_t kvs_evict_attn_bwd_workspace(int B, int T, int Hq, int Hkv, int D) {
  if (B < 1 || T < 1 || Hq < 1 || Hkv < 1) return 0;
  return bwd_ws(B, T, (long long)B * T, Hq, Hkv, D);
}

size_t kvs_evict_attn_varlen_fwd_workspace(int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D) {
  if (B < 1 || Ntot < 0) return 0;
  (void)max_seqlen; (void)Hq; (void)Hkv; (void)D;
  return fwd_ws(B, Ntot);
}

size_t kvs_evict_attn_varlen_bwd_workspace(int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D) {
  if (B < 1 || Ntot < 0 || Hq < 1 || Hkv < 1 || max_seqlen < 1) return 0;
  return bwd_ws(B, max_seqlen, Ntot, Hq, Hkv, D);
}

constexpr unsigned kKnownFlags = KVS_FLAG_NO_EMPTY_SKIP | KVS_FLAG_FULL_AS_PARTIAL;

static kvs_status_t fwd_common(const void* Q, const void* K, const void* V, const int32_t* evict_at,
                               const int32_t* cu, void* O, float* LSE, int B, int T, long long ntok, int Hq,
                               int Hkv, int D, float scale, unsigned flags, void* ws, size_t ws_bytes,
                               void* stream) {
  t_err.clear();
  kvs_status_t st = check_dims(B, T, ntok, Hq, Hkv, D);
  if (st != KVS_OK) return st;
  if (!(scale > 0.f) || scale != scale) return fail(KVS_ERR_SHAPE, "softmax_scale must be positive and finite");
  if (flags & ~kKnownFlags) return fail(KVS_ERR_UNSUPPORTED, "unknown flag bits 0x%x", flags & ~kKnownFlags);
  // An empty batch has nothing to read or write: its pointers (zero-size
  // buffers, possibly NULL) and workspace are not looked at.
  if (ntok == 0) return KVS_OK;
  REQUIRE_PTR(Q, "Q");
  REQUIRE_PTR(K, "K");
  REQUIRE_PTR(V, "V");
  REQUIRE_PTR(O, "O");
  REQUIRE_PTR(LSE, "LSE");
  if (!evict_at) return fail(KVS_ERR_NULL, "evict_at is NULL");
  st = check_ws(ws, ws_bytes, fwd_ws(B, ntok));
  if (st != KVS_OK) return st;
  kvs::Problem p{};
  p.q = Q; p.k = K; p.v = V; p.evict = evict_at; p.cu = cu; p.o = O; p.lse = LSE;
  p.B = B; p.T = T; p.ntok = (int)ntok; p.Hq = Hq; p.Hkv = Hkv; p.D = D; p.G = Hq / Hkv;
  p.flags = (int)flags; p.scale = scale; p.ws = ws; p.stream = (hipStream_t)stream;
  return run_fwd(p);
}

static kvs_status_t bwd_common(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                               const float* LSE, const int32_t* evict_at, const int32_t* cu, void* dQ, void* dK,
                               void* dV, int B, int T, long long ntok, int Hq, int Hkv, int D, float scale,
                               unsigned flags, void* ws, size_t ws_bytes, void* stream) {
  t_err.clear();
  kvs_status_t st = check_dims(B, T, ntok, Hq, Hkv, D);
  if (st != KVS_OK) return st;
  if (!(scale > 0.f) || scale != scale) return fail(KVS_ERR_SHAPE, "softmax_scale must be positive and finite");
  if (flags & ~kKnownFlags) return fail(KVS_ERR_UNSUPPORTED, "unknown flag bits 0x%x", flags & ~kKnownFlags);
  if (ntok == 0) return KVS_OK;  // empty batch: pointers and workspace are not looked at
  REQUIRE_PTR(dO, "dO");
  REQUIRE_PTR(Q, "Q");
  REQUIRE_PTR(K, "K");
  REQUIRE_PTR(V, "V");
  REQUIRE_PTR(O, "O");
  REQUIRE_PTR(LSE, "LSE");
  REQUIRE_PTR(dQ, "dQ");
  REQUIRE_PTR(dK, "dK");
  REQUIRE_PTR(dV, "dV");
  if (!evict_at) return fail(KVS_ERR_NULL, "evict_at is NULL");
  st = check_ws(ws, ws_bytes, bwd_ws(B, T, ntok, Hq, Hkv, D));
  if (st != KVS_OK) return st;
  kvs::Problem p{};
  p.q = Q; p.k = K; p.v = V; p.o_in = O; p.dout = dO; p.lse_in = LSE; p.evict = evict_at; p.cu = cu;
  p.dq = dQ; p.dk = dK; p.dv = dV;
  p.B = B; p.T = T; p.ntok = (int)ntok; p.Hq = Hq; p.Hkv = Hkv; p.D = D; p.G = Hq / Hkv;
  p.flags = (int)flags; p.scale = scale; p.ws = ws; p.stream = (hipStream_t)stream;
  return run_bwd(p);
}

kvs_status_t kvs_evict_attn_fwd(const void* Q, const void* K, const void* V, const int32_t* evict_at, void* O,
                                float* LSE, int B, int T, int Hq, int Hkv, int D, float softmax_scale,
                                void* workspace, size_t workspace_bytes, void* stream) {
  return fwd_common(Q, K, V, evict_at, nullptr, O, LSE, B, T, (long long)B * T, Hq, Hkv, D, softmax_scale, 0u,
                    workspace, workspace_bytes, stream);
}

kvs_status_t kvs_evict_attn_bwd(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                                const float* LSE, const int32_t* evict_at, void* dQ, void* dK, void* dV, int B,
                                int T, int Hq, int Hkv, int D, float softmax_scale, void* workspace,
                                size_t workspace_bytes, void* stream) {
  return bwd_common(dO, Q, K, V, O, LSE, evict_at, nullptr, dQ, dK, dV, B, T, (long long)B * T, Hq, Hkv, D,
                    softmax_scale, 0u, workspace, workspace_bytes, stream);
}

kvs_status_t kvs_evict_attn_varlen_fwd(const void* Q, const void* K, const void* V, const int32_t* evict_at,
                                       const int32_t* cu_seqlens, void* O, float* LSE, int B, int Ntot,
                                       int max_seqlen, int Hq, int Hkv, int D, float softmax_scale, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  if (!cu_seqlens) return fail(KVS_ERR_NULL, "cu_seqlens is NULL");
  return fwd_common(Q, K, V, evict_at, cu_seqlens, O, LSE, B, max_seqlen, Ntot, Hq, Hkv, D, softmax_scale, 0u,
                    workspace, workspace_bytes, stream);
}

kvs_status_t kvs_evict_attn_varlen_bwd(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                                       const float* LSE, const int32_t* evict_at, const int32_t* cu_seqlens,
                                       void* dQ, void* dK, void* dV, int B, int Ntot, int max_seqlen, int Hq,
                                       int Hkv, int D, float softmax_scale, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  if (!cu_seqlens) return fail(KVS_ERR_NULL, "cu_seqlens is NULL");
  return bwd_common(dO, Q, K, V, O, LSE, evict_at, cu_seqlens, dQ, dK, dV, B, max_seqlen, Ntot, Hq, Hkv, D,
                    softmax_scale, 0u, workspace, workspace_bytes, stream);
}

// Fixed length (cu_seqlens NULL: B traces of max_seqlen tokens, Ntot = B * max_seqlen) or varlen, with
// the tile-classifier switches.
static kvs_status_t ex_dims(const int32_t* cu, int B, int Ntot, int max_seqlen) {
  if (!cu && (long long)B * max_seqlen != (long long)Ntot)
    return fail(KVS_ERR_SHAPE, "without cu_seqlens, Ntot (%d) must equal B * max_seqlen (%d * %d)", Ntot, B,
                max_seqlen);
  return KVS_OK;
}

kvs_status_t kvs_evict_attn_fwd_ex(const void* Q, const void* K, const void* V, const int32_t* evict_at,
                                   const int32_t* cu_seqlens, void* O, float* LSE, int B, int Ntot, int max_seqlen,
                                   int Hq, int Hkv, int D, float softmax_scale, unsigned flags, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  t_err.clear();
  if (kvs_status_t st = ex_dims(cu_seqlens, B, Ntot, max_seqlen)) return st;
  return fwd_common(Q, K, V, evict_at, cu_seqlens, O, LSE, B, max_seqlen, Ntot, Hq, Hkv, D, softmax_scale, flags,
                    workspace, workspace_bytes, stream);
}

kvs_status_t kvs_evict_attn_bwd_ex(const void* dO, const void* Q, const void* K, const void* V, const void* O,
                                   const float* LSE, const int32_t* evict_at, const int32_t* cu_seqlens, void* dQ,
                                   void* dK, void* dV, int B, int Ntot, int max_seqlen, int Hq, int Hkv, int D,
                                   float softmax_scale, unsigned flags, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  t_err.clear();
  if (kvs_status_t st = ex_dims(cu_seqlens, B, Ntot, max_seqlen)) return st;
  return bwd_common(dO, Q, K, V, O, LSE, evict_at, cu_seqlens, dQ, dK, dV, B, max_seqlen, Ntot, Hq, Hkv, D,
                    softmax_scale, flags, workspace, workspace_bytes, stream);
}

kvs_status_t kvs_evict_attn_fwd_noalloc(const void* Q, const void* K, const void* V, const int32_t* evict_at,
                                        const int32_t* cu_seqlens, void* O, float* LSE, int B, int Ntot,
                                        int max_seqlen, int Hq, int Hkv, int D, float softmax_scale, void* stream) {
  t_err.clear();
  if (kvs_status_t st = ex_dims(cu_seqlens, B, Ntot, max_seqlen)) return st;
  if (kvs_status_t st = check_dims(B, max_seqlen, Ntot, Hq, Hkv, D)) return st;
  const size_t need = fwd_ws(B, Ntot);
  if (need > kvs::kNoAllocScratchBytes)
    return fail(KVS_ERR_UNSUPPORTED, "allocation-free forward: %zu bytes of scratch needed, %zu available "
                "(B + Ntot / 64 + 2 must stay within %zu key tiles)", need, kvs::kNoAllocScratchBytes,
                kvs::kNoAllocScratchBytes / 8);
  if (!(softmax_scale > 0.f) || softmax_scale != softmax_scale)
    return fail(KVS_ERR_SHAPE, "softmax_scale must be positive and finite");
  if (Ntot == 0) return KVS_OK;  // empty batch: pointers are not looked at
  REQUIRE_PTR(Q, "Q");
  REQUIRE_PTR(K, "K");
  REQUIRE_PTR(V, "V");
  REQUIRE_PTR(O, "O");
  REQUIRE_PTR(LSE, "LSE");
  if (!evict_at) return fail(KVS_ERR_NULL, "evict_at is NULL");
  void* scratch = nullptr;
  hipError_t e = kvs::noalloc_scratch(&scratch);
  if (e != hipSuccess) return hip_fail(e, "device address of the library scratch");
  return fwd_common(Q, K, V, evict_at, cu_seqlens, O, LSE, B, max_seqlen, Ntot, Hq, Hkv, D, softmax_scale, 0u,
                    scratch, kvs::kNoAllocScratchBytes, stream);
}

kvs_status_t kvs_classify_tiles(const int32_t* evict_at, const int32_t* cu_seqlens, int B, int T, int BM, int BN,
                                uint8_t* tile_class, void* stream) {
  t_err.clear();
  if (B < 1 || T < 1) return fail(KVS_ERR_SHAPE, "B and T must be >= 1");
  if (T > kMaxSeq * 16) return fail(KVS_ERR_UNSUPPORTED, "T above %d", kMaxSeq * 16);
  if (BM < 16 || BM > 256 || BM % 16 != 0) return fail(KVS_ERR_SHAPE, "BM must be a multiple of 16 in [16, 256]");
  if (BN != 32 && BN != 64 && BN != 128) return fail(KVS_ERR_SHAPE, "BN must be 32, 64 or 128");
  if (!evict_at) return fail(KVS_ERR_NULL, "evict_at is NULL");
  if (!tile_class) return fail(KVS_ERR_NULL, "tile_class is NULL");
  hipError_t e = kvs::launch_classify(evict_at, cu_seqlens, B, T, BM, BN, tile_class, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "classify launch");
  return KVS_OK;
}

size_t kvs_classify_tiles_size(const int32_t* lengths, int B, int BM, int BN) {
  if (!lengths || B < 1 || BM < 1 || BN < 1) return 0;
  size_t n = 0;
  for (int b = 0; b < B; ++b) {
    const long long L = lengths[b] > 0 ? lengths[b] : 0;
    n += (size_t)((L + BM - 1) / BM) * (size_t)((L + BN - 1) / BN);
  }
  return n;
}

kvs_status_t kvs_check_evict_at(const int32_t* evict_at, const int32_t* cu_seqlens, int B, int T,
                                int64_t* first_bad, void* stream) {
  t_err.clear();
  if (!first_bad) return fail(KVS_ERR_NULL, "first_bad is NULL");
  *first_bad = -1;
  if (B < 1 || T < 0) return fail(KVS_ERR_SHAPE, "B must be >= 1 and T >= 0");
  if (!evict_at) return fail(KVS_ERR_NULL, "evict_at is NULL");
  const long long ntok = cu_seqlens ? T : (long long)B * T;
  if (ntok > 0x7fffffffll) return fail(KVS_ERR_UNSUPPORTED, "too many tokens");
  int cu_bad = 0;
  std::lock_guard<std::mutex> lk(g_check_mu);
  hipError_t e = kvs::launch_check(evict_at, cu_seqlens, B, T, (int)ntok, first_bad, &cu_bad, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "evict_at check");
  if (cu_bad) return fail(KVS_ERR_SHAPE, "cu_seqlens is not 0 = cu[0] <= ... <= cu[B] = Ntot");
  if (*first_bad >= 0) return fail(KVS_ERR_EVICT, "evict_at[%lld] <= its local index", (long long)*first_bad);
  return KVS_OK;
}

void kvs_prof_enable(int on) { g_prof.store(on != 0); }

void kvs_prof_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  g_recs.clear();
}

kvs_status_t kvs_prof_read(const char* name, int* launches, double* total_ms) {
  t_err.clear();
  if (!name || !launches || !total_ms) return fail(KVS_ERR_NULL, "NULL argument");
  int n = 0;
  double tot = 0.0;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_recs) {
    if (std::strcmp(r.name, name) != 0) continue;
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return hip_fail(e, "event synchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return hip_fail(e, "event elapsed time");
    ++n;
    tot += ms;
  }
  *launches = n;
  *total_ms = tot;
  return KVS_OK;
}

// ---------------------------------------------------------------- streamed paged KV cache
struct kvs_block_manager {
  kvs::BlockManager impl;
};

static kvs_status_t bm_status(int code, const std::string& msg) {
  switch (code) {
    case kvs::BlockManager::kOk: return KVS_OK;
    case kvs::BlockManager::kBadArg: return fail(KVS_ERR_SHAPE, "%s", msg.c_str());
    case kvs::BlockManager::kBadState: return fail(KVS_ERR_STATE, "%s", msg.c_str());
    default: return fail(KVS_ERR_CAPACITY, "%s", msg.c_str());
  }
}

kvs_status_t kvs_bm_create(int num_blocks, int block_size, int num_seqs, int max_blocks, kvs_block_manager** out) {
  t_err.clear();
  if (!out) return fail(KVS_ERR_NULL, "out is NULL");
  *out = nullptr;
  if (num_blocks < 1 || block_size < 1 || num_seqs < 1 || max_blocks < 1)
    return fail(KVS_ERR_SHAPE, "num_blocks, block_size, num_seqs, max_blocks must be >= 1");
  if (block_size > 64) return fail(KVS_ERR_SHAPE, "block_size %d above 64", block_size);
  if ((long long)num_blocks * block_size > 0x7fffffffll)
    return fail(KVS_ERR_UNSUPPORTED, "num_blocks * block_size above INT32_MAX");
  *out = new kvs_block_manager{kvs::BlockManager(num_blocks, block_size, num_seqs, max_blocks)};
  return KVS_OK;
}

void kvs_bm_destroy(kvs_block_manager* bm) { delete bm; }

kvs_status_t kvs_bm_append(kvs_block_manager* bm, int seq, const int32_t* pos, int n, int32_t* slots) {
  t_err.clear();
  if (!bm) return fail(KVS_ERR_NULL, "block manager is NULL");
  if (n < 0) return fail(KVS_ERR_SHAPE, "n must be >= 0");
  if (n > 0 && (!pos || !slots)) return fail(KVS_ERR_NULL, "pos or slots is NULL");
  std::string msg;
  return bm_status(bm->impl.append(seq, pos, n, slots, &msg), msg);
}

kvs_status_t kvs_bm_evict(kvs_block_manager* bm, int seq, const int32_t* pos, int n, int32_t* slots) {
  t_err.clear();
  if (!bm) return fail(KVS_ERR_NULL, "block manager is NULL");
  if (n < 0) return fail(KVS_ERR_SHAPE, "n must be >= 0");
  if (n > 0 && (!pos || !slots)) return fail(KVS_ERR_NULL, "pos or slots is NULL");
  std::string msg;
  return bm_status(bm->impl.evict(seq, pos, n, slots, &msg), msg);
}

kvs_status_t kvs_bm_release(kvs_block_manager* bm, int seq, int32_t* slots, int* n_slots) {
  t_err.clear();
  if (!bm || !n_slots) return fail(KVS_ERR_NULL, "block manager or n_slots is NULL");
  if (bm->impl.live(seq) > 0 && !slots) return fail(KVS_ERR_NULL, "slots is NULL");
  std::string msg;
  return bm_status(bm->impl.release(seq, slots, n_slots, &msg), msg);
}

kvs_status_t kvs_bm_tables(const kvs_block_manager* bm, int32_t* block_table, int32_t* seq_blocks) {
  t_err.clear();
  if (!bm || !block_table || !seq_blocks) return fail(KVS_ERR_NULL, "NULL argument");
  bm->impl.tables(block_table, seq_blocks);
  return KVS_OK;
}

int kvs_bm_free_blocks(const kvs_block_manager* bm) { return bm ? bm->impl.free_blocks() : -1; }
int kvs_bm_live(const kvs_block_manager* bm, int seq) { return bm ? bm->impl.live(seq) : -1; }

static kvs_status_t check_cache_dims(int num_blocks, int block_size) {
  if (num_blocks < 1 || block_size < 1 || block_size > 64)
    return fail(KVS_ERR_SHAPE, "num_blocks must be >= 1 and block_size in [1, 64]");
  if ((long long)num_blocks * block_size > 0x7fffffffll)
    return fail(KVS_ERR_UNSUPPORTED, "num_blocks * block_size above INT32_MAX");
  return KVS_OK;
}

kvs_status_t kvs_paged_append(const void* K_new, const void* V_new, const int32_t* positions, const int32_t* slots,
                              int n, void* K_cache, void* V_cache, int32_t* slot_pos, int num_blocks,
                              int block_size, int Hkv, int D, void* stream) {
  t_err.clear();
  if (kvs_status_t st = check_cache_dims(num_blocks, block_size)) return st;
  if (n < 0 || Hkv < 1) return fail(KVS_ERR_SHAPE, "n must be >= 0 and Hkv >= 1");
  if (D != 64 && D != 128) return fail(KVS_ERR_SHAPE, "head dim D must be 64 or 128 (got %d)", D);
  REQUIRE_PTR(K_cache, "K_cache");
  REQUIRE_PTR(V_cache, "V_cache");
  if (!slot_pos) return fail(KVS_ERR_NULL, "slot_pos is NULL");
  if (n == 0) return KVS_OK;
  REQUIRE_PTR(K_new, "K_new");
  REQUIRE_PTR(V_new, "V_new");
  if (!positions || !slots) return fail(KVS_ERR_NULL, "positions or slots is NULL");
  hipError_t e = kvs::launch_paged_append(K_new, V_new, positions, slots, n, K_cache, V_cache, slot_pos,
                                          num_blocks * block_size, block_size, Hkv, D, (hipStream_t)stream);
  return e == hipSuccess ? KVS_OK : hip_fail(e, "paged append launch");
}

kvs_status_t kvs_paged_evict(const int32_t* slots, int n, int32_t* slot_pos, int num_blocks, int block_size,
                             void* stream) {
  t_err.clear();
  if (kvs_status_t st = check_cache_dims(num_blocks, block_size)) return st;
  if (n < 0) return fail(KVS_ERR_SHAPE, "n must be >= 0");
  if (!slot_pos) return fail(KVS_ERR_NULL, "slot_pos is NULL");
  if (n == 0) return KVS_OK;
  if (!slots) return fail(KVS_ERR_NULL, "slots is NULL");
  hipError_t e = kvs::launch_paged_evict(slots, n, slot_pos, num_blocks * block_size, (hipStream_t)stream);
  return e == hipSuccess ? KVS_OK : hip_fail(e, "paged evict launch");
}

static kvs_status_t check_decode_dims(int S, int Hq, int Hkv, int D, int num_blocks, int block_size,
                                      int max_blocks) {
  if (S < 1 || Hq < 1 || Hkv < 1 || max_blocks < 1)
    return fail(KVS_ERR_SHAPE, "num_seqs, Hq, Hkv, max_blocks must be >= 1");
  if (Hq % Hkv != 0) return fail(KVS_ERR_SHAPE, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
  if (D != 64 && D != 128) return fail(KVS_ERR_SHAPE, "head dim D must be 64 or 128 (got %d)", D);
  if (kvs_status_t st = check_cache_dims(num_blocks, block_size)) return st;
  if (Hq / Hkv > 32) return fail(KVS_ERR_UNSUPPORTED, "decode supports GQA groups of at most 32 (got %d)", Hq / Hkv);
  if ((long long)max_blocks * block_size > 0x7fffffffll)
    return fail(KVS_ERR_UNSUPPORTED, "max_blocks * block_size above INT32_MAX");
  if ((long long)S * Hkv * kvs::paged_nsplit(S, Hkv, max_blocks, block_size, D) > 0x7fffffffll)
    return fail(KVS_ERR_UNSUPPORTED, "decode grid too large");
  return KVS_OK;
}

size_t kvs_paged_decode_workspace(int num_seqs, int Hq, int Hkv, int D, int max_blocks, int block_size) {
  if (num_seqs < 1 || Hkv < 1 || max_blocks < 1 || block_size < 1) return 0;
  return kvs::paged_ws_bytes(num_seqs, Hq, D, kvs::paged_nsplit(num_seqs, Hkv, max_blocks, block_size, D));
}

kvs_status_t kvs_paged_decode(const void* Q, const void* K_cache, const void* V_cache, const int32_t* slot_pos,
                              const int32_t* block_table, const int32_t* seq_blocks, void* O, float* LSE,
                              int num_seqs, int Hq, int Hkv, int D, int num_blocks, int block_size, int max_blocks,
                              float softmax_scale, void* workspace, size_t workspace_bytes, void* stream) {
  t_err.clear();
  if (kvs_status_t st = check_decode_dims(num_seqs, Hq, Hkv, D, num_blocks, block_size, max_blocks)) return st;
  if (!(softmax_scale > 0.f) || softmax_scale != softmax_scale)
    return fail(KVS_ERR_SHAPE, "softmax_scale must be positive and finite");
  REQUIRE_PTR(Q, "Q");
  REQUIRE_PTR(K_cache, "K_cache");
  REQUIRE_PTR(V_cache, "V_cache");
  REQUIRE_PTR(O, "O");
  if (!slot_pos || !block_table || !seq_blocks || !LSE) return fail(KVS_ERR_NULL, "NULL table or output pointer");
  const size_t need = kvs_paged_decode_workspace(num_seqs, Hq, Hkv, D, max_blocks, block_size);
  if (kvs_status_t st = check_ws(workspace, workspace_bytes, need)) return st;
  kvs::PagedDecode p{};
  p.q = Q;
  p.k_cache = K_cache;
  p.v_cache = V_cache;
  p.slot_pos = slot_pos;
  p.block_table = block_table;
  p.seq_blocks = seq_blocks;
  p.o = O;
  p.lse = LSE;
  p.S = num_seqs;
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.D = D;
  p.max_blocks = max_blocks;
  p.block_size = block_size;
  p.num_blocks = num_blocks;
  p.scale = softmax_scale;
  p.ws = workspace;
  p.stream = (hipStream_t)stream;
  hipError_t e = kvs::launch_paged_decode(p);
  return e == hipSuccess ? KVS_OK : hip_fail(e, "paged decode launch");
}

}  // extern "C"
