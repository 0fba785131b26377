// C ABI of the aTTT update-step library: argument validation (host only, before any HIP
// call), workspace planning, episode / problem batching into kernel-argument descriptors,
// kernel launches on the caller's stream, and optional per-kernel event timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "attt.h"
#include "internal.hpp"

using namespace attt;

static_assert(kNgramScratchBytes == ATTT_NGRAM_NOALLOC_SCRATCH_BYTES, "header and library agree on the scratch size");

// ------------------------------------------------------------------------------------------
// Status, messages, timing registry
// ------------------------------------------------------------------------------------------
static thread_local std::string g_last_error;

static attt_status fail(attt_status code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
static attt_status fail(attt_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

static attt_status hip_fail(hipError_t e, const char* where) {
  return fail(ATTT_EHIP, "%s: %s", where, hipGetErrorString(e));
}

#define HIP_TRY(expr, where)                  \
  do {                                        \
    hipError_t e_ = (expr);                   \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

namespace attt {

static const char* kKernelNames[K_NUM_KERNELS] = {
    "ngram_count", "ngram_weight", "ngram_table", "ce_fwd_lse", "ce_label_logit", "ce_row_reduce",
    "ce_loss", "ce_head_transpose", "ce_bwd_dz", "ce_bwd_dh", "ce_overflow_guard", "lora_u_du", "lora_dadb",
    "lora_reduce", "ngram_set", "ngram_set_weight", "lora_sgd", "ce_fused_bwd", "rep_count", "rep_reduce", "attn_fwd_stats",
    "attn_dkdv", "attn_dq", "lora_fwd", "lora_swap"};

const char* kernel_name(int id) { return (id >= 0 && id < K_NUM_KERNELS) ? kKernelNames[id] : nullptr; }

struct TimingRec {
  int id;
  hipEvent_t a, b;
};
static std::mutex g_tmu;
static bool g_timing = false;
static std::vector<TimingRec> g_recs;
static double g_ms[K_NUM_KERNELS];
static int64_t g_launches[K_NUM_KERNELS];

bool timing_on() { return g_timing; }

void timing_record(int id, hipEvent_t a, hipEvent_t b) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_recs.push_back({id, a, b});
}

static hipError_t timing_drain() {
  hipError_t first = hipSuccess;
  for (auto& r : g_recs) {
    hipError_t e = hipEventSynchronize(r.b);
    float ms = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e == hipSuccess) {
      g_ms[r.id] += ms;
      g_launches[r.id] += 1;
    } else if (first == hipSuccess) {
      first = e;
    }
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  g_recs.clear();
  return first;
}

}  // namespace attt

extern "C" {

const char* attt_status_string(attt_status s) {
  switch (s) {
    case ATTT_OK: return "ok";
    case ATTT_EINVAL: return "invalid argument";
    case ATTT_ENOSPACE: return "workspace too small";
    case ATTT_EUNSUPPORTED: return "unsupported by this build";
    case ATTT_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* attt_last_error(void) { return g_last_error.c_str(); }

int32_t attt_version(void) { return 100; }

attt_status attt_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
  return ATTT_OK;
}

attt_status attt_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_tmu);
  hipError_t e = timing_drain();
  std::fill(g_ms, g_ms + K_NUM_KERNELS, 0.0);
  std::fill(g_launches, g_launches + K_NUM_KERNELS, 0);
  if (e != hipSuccess) return hip_fail(e, "attt_timing_reset");
  return ATTT_OK;
}

attt_status attt_timing_read(const char* kernel, double* total_ms, int64_t* launches) {
  if (!kernel || !total_ms || !launches) return fail(ATTT_EINVAL, "attt_timing_read: null argument");
  int id = -1;
  for (int i = 0; i < K_NUM_KERNELS; ++i)
    if (std::strcmp(kernel, kKernelNames[i]) == 0) id = i;
  if (id < 0) return fail(ATTT_EINVAL, "attt_timing_read: unknown kernel '%s'", kernel);
  std::lock_guard<std::mutex> lk(g_tmu);
  hipError_t e = timing_drain();
  if (e != hipSuccess) return hip_fail(e, "attt_timing_read");
  *total_ms = g_ms[id];
  *launches = g_launches[id];
  return ATTT_OK;
}

const char* attt_timing_kernel_name(int32_t i) { return kernel_name(i); }

}  // extern "C"

// ------------------------------------------------------------------------------------------
// Helpers
// ------------------------------------------------------------------------------------------
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
static inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
static inline bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

static attt_status check_offsets(const char* what, const int64_t* off, int32_t E, int64_t limit) {
  if (!off) return fail(ATTT_EINVAL, "%s: offsets pointer is null", what);
  if (off[0] != 0) return fail(ATTT_EINVAL, "%s: offsets[0] must be 0", what);
  for (int32_t e = 0; e < E; ++e) {
    if (off[e + 1] < off[e]) return fail(ATTT_EINVAL, "%s: offsets decrease at episode %d", what, e);
    if (off[e + 1] - off[e] > limit)
      return fail(ATTT_EUNSUPPORTED, "%s: episode %d holds %lld entries (limit %lld)", what, e,
                  (long long)(off[e + 1] - off[e]), (long long)limit);
  }
  return ATTT_OK;
}

// ------------------------------------------------------------------------------------------
// n-gram exposure and weights
// ------------------------------------------------------------------------------------------
namespace {

struct NgramEpPlan {
  int64_t tok_base, hist_base, chunk_base, part_base;
  int32_t L, Q, hist_ngrams, parts, chunks;
};

// workspace: partial counts [total_chunks][kQMax] u16, then canon [total_parts][kQMax] u16, then
// list [total_parts][kQMax] uint2
struct NgramPlan {
  std::vector<NgramEpPlan> eps;
  int64_t total_chunks = 0, total_parts = 0;
  size_t off_canon = 0, off_list = 0;
  size_t total = 0;
};

int next_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

attt_status ngram_validate(const int64_t* hoff, const int64_t* toff, int32_t E, int32_t n) {
  if (E < 1) return fail(ATTT_EINVAL, "ngram: num_episodes must be >= 1 (got %d)", E);
  if (n < 1 || n > ATTT_NGRAM_MAX_N)
    return fail(ATTT_EINVAL, "ngram: n must be in [1, %d] (got %d)", ATTT_NGRAM_MAX_N, n);
  attt_status st = check_offsets("ngram history", hoff, E, INT32_MAX);
  if (st) return st;
  st = check_offsets("ngram tokens", toff, E, INT32_MAX);
  if (st) return st;
  if (toff[E] >= ((int64_t)1 << 31)) return fail(ATTT_EUNSUPPORTED, "ngram: more than 2^31-1 update tokens");
  return ATTT_OK;
}

// History chunks: about two workgroups per CU over the whole call, at most 65535 positions
// per chunk (the per-chunk counts are 16-bit) and at least 2048.
NgramPlan ngram_plan(const int64_t* hoff, const int64_t* toff, int32_t E, int32_t n) {
  NgramPlan P;
  int64_t work = 0;
  for (int32_t e = 0; e < E; ++e) {
    const int64_t L = toff[e + 1] - toff[e], H = hoff[e + 1] - hoff[e];
    const int64_t Q = std::max<int64_t>(0, L - n + 1);
    work += ceil_div(Q, kQMax) * std::max<int64_t>(0, H - n + 1);
  }
  // one count workgroup per CU (its LDS table takes most of the CU): about 256 chunks in all,
  // so every workgroup sets its table up once
  const int64_t chunk_len = std::min<int64_t>(65535, std::max<int64_t>(2048, ceil_div(work, 256)));
  for (int32_t e = 0; e < E; ++e) {
    NgramEpPlan ep{};
    ep.tok_base = toff[e];
    ep.hist_base = hoff[e];
    ep.L = (int32_t)(toff[e + 1] - toff[e]);
    ep.Q = std::max(0, ep.L - n + 1);
    ep.hist_ngrams = (int32_t)std::max<int64_t>(0, hoff[e + 1] - hoff[e] - n + 1);
    ep.parts = (int32_t)ceil_div(ep.Q, kQMax);
    ep.chunks = ep.hist_ngrams > 0 ? (int32_t)ceil_div(ep.hist_ngrams, chunk_len) : 0;
    ep.chunk_base = P.total_chunks;
    ep.part_base = P.total_parts;
    P.total_chunks += (int64_t)ep.parts * ep.chunks;
    if (ep.chunks > 0) P.total_parts += ep.parts;
    P.eps.push_back(ep);
  }
  P.off_canon = align256((size_t)P.total_chunks * kQMax * 2);
  P.off_list = P.off_canon + align256((size_t)P.total_parts * kQMax * 2);
  P.total = std::max<size_t>(P.off_list + align256((size_t)P.total_parts * kQMax * 8), 256);
  return P;
}

}  // namespace

extern "C" attt_status attt_ngram_workspace_size(const int64_t* history_offsets,
                                                 const int64_t* token_offsets, int32_t num_episodes,
                                                 int32_t n, size_t* bytes) {
  if (!bytes) return fail(ATTT_EINVAL, "ngram: bytes is null");
  attt_status st = ngram_validate(history_offsets, token_offsets, num_episodes, n);
  if (st) return st;
  *bytes = ngram_plan(history_offsets, token_offsets, num_episodes, n).total;
  return ATTT_OK;
}

namespace {
attt_status ngram_check_args(const int32_t* history, const int64_t* history_offsets, const int32_t* tokens,
                             const int64_t* token_offsets, int32_t num_episodes, int32_t n, float w_min,
                             float* weights) {
  attt_status st = ngram_validate(history_offsets, token_offsets, num_episodes, n);
  if (st) return st;
  if (!(w_min >= 0x1p-20f && w_min <= 1.0f))
    return fail(ATTT_EINVAL, "ngram: w_min must be in [2^-20, 1] (got %g)", (double)w_min);
  const int64_t T = token_offsets[num_episodes];
  if (T > 0 && !tokens) return fail(ATTT_EINVAL, "ngram: tokens is null");
  if (T > 0 && !weights) return fail(ATTT_EINVAL, "ngram: weights is null");
  if (history_offsets[num_episodes] > 0 && !history) return fail(ATTT_EINVAL, "ngram: history is null");
  return ATTT_OK;
}

attt_status ngram_run(const NgramPlan& P, const int32_t* history, const int32_t* tokens, int32_t E,
                      int32_t n, float w_min, uint32_t* exposure, float* weights, void* workspace,
                      hipStream_t s);
}  // namespace

extern "C" attt_status attt_ngram_weights(const int32_t* history, const int64_t* history_offsets,
                                          const int32_t* tokens, const int64_t* token_offsets,
                                          int32_t num_episodes, int32_t n, float w_min,
                                          uint32_t* exposure, float* weights, void* workspace,
                                          size_t workspace_bytes, void* stream) {
  attt_status st = ngram_check_args(history, history_offsets, tokens, token_offsets, num_episodes, n, w_min,
                                    weights);
  if (st) return st;
  NgramPlan P = ngram_plan(history_offsets, token_offsets, num_episodes, n);
  if (workspace_bytes < P.total)
    return fail(ATTT_ENOSPACE, "ngram: workspace %zu bytes, need %zu", workspace_bytes, P.total);
  if (!workspace) return fail(ATTT_EINVAL, "ngram: workspace is null");
  if (!aligned256(workspace)) return fail(ATTT_EINVAL, "ngram: workspace must be 256-byte aligned");
  if (token_offsets[num_episodes] == 0) return ATTT_OK;
  return ngram_run(P, history, tokens, num_episodes, n, w_min, exposure, weights, workspace,
                   static_cast<hipStream_t>(stream));
}

extern "C" attt_status attt_ngram_weights_noalloc(const int32_t* history, const int64_t* history_offsets,
                                                  const int32_t* tokens, const int64_t* token_offsets,
                                                  int32_t num_episodes, int32_t n, float w_min,
                                                  uint32_t* exposure, float* weights, void* stream) {
  attt_status st = ngram_check_args(history, history_offsets, tokens, token_offsets, num_episodes, n, w_min,
                                    weights);
  if (st) return st;
  NgramPlan P = ngram_plan(history_offsets, token_offsets, num_episodes, n);
  if (P.total > kNgramScratchBytes)
    return fail(ATTT_EUNSUPPORTED,
                "ngram_noalloc: the call needs %zu bytes of scratch, beyond the static %zu-byte buffer "
                "(use attt_ngram_weights with a workspace)", P.total, kNgramScratchBytes);
  if (token_offsets[num_episodes] == 0) return ATTT_OK;
  void* scratch = nullptr;
  HIP_TRY(ngram_scratch(&scratch), "ngram_noalloc: scratch address");
  return ngram_run(P, history, tokens, num_episodes, n, w_min, exposure, weights, scratch,
                   static_cast<hipStream_t>(stream));
}

namespace {
attt_status ngram_run(const NgramPlan& P, const int32_t* history, const int32_t* tokens, int32_t E,
                      int32_t n, float w_min, uint32_t* exposure, float* weights, void* workspace,
                      hipStream_t s) {

  uint16_t* partial = static_cast<uint16_t*>(workspace);
  uint16_t* canon = reinterpret_cast<uint16_t*>(static_cast<uint8_t*>(workspace) + P.off_canon);
  uint2* list = reinterpret_cast<uint2*>(static_cast<uint8_t*>(workspace) + P.off_list);

  // table and count kernels: batches of partitions; a partition's chunks are consecutive
  // count-kernel blocks
  NgramPartBatch batch{};
  int blocks = 0, max_slots = 64;
  auto flush = [&]() -> attt_status {
    if (batch.count == 0) return ATTT_OK;
    HIP_TRY(launch_ngram_table(batch, max_slots, tokens, n, canon, list, s), "ngram_table");
    HIP_TRY(launch_ngram_count(batch, blocks, max_slots, history, tokens, list, n, partial, s), "ngram_count");
    batch = NgramPartBatch{};
    blocks = 0;
    max_slots = 64;
    return ATTT_OK;
  };
  for (const auto& ep : P.eps) {
    if (ep.chunks == 0) continue;
    for (int32_t p = 0; p < ep.parts; ++p) {
      if (batch.count == kPartBatch) {
        attt_status st2 = flush();
        if (st2) return st2;
      }
      NgramPart& q = batch.p[batch.count++];
      q.tok_base = ep.tok_base;
      q.hist_base = ep.hist_base;
      q.hist_ngrams = ep.hist_ngrams;
      q.q0 = p * kQMax;
      q.qn = std::min(kQMax, ep.Q - p * kQMax);
      q.slots = std::max(64, next_pow2(8 * q.qn));  // load factor <= 1/8: a second bucket is rare
      q.chunks = ep.chunks;
      q.chunk_begin = blocks;
      q.chunk_begin_global = ep.chunk_base + (int64_t)p * ep.chunks;
      q.part_global = ep.part_base + p;
      blocks += ep.chunks;
      max_slots = std::max(max_slots, q.slots);
    }
  }
  {
    attt_status st2 = flush();
    if (st2) return st2;
  }
  for (int32_t e0 = 0; e0 < E; e0 += kEpBatch) {
    NgramEpBatch wb{};
    wb.count = std::min<int32_t>(kEpBatch, E - e0);
    int wblocks = 0;
    for (int i = 0; i < wb.count; ++i) {
      const NgramEpPlan& ep = P.eps[e0 + i];
      wb.e[i].tok_base = ep.tok_base;
      wb.e[i].chunk_base = ep.chunk_base;
      wb.e[i].part_base = ep.part_base;
      wb.e[i].L = ep.L;
      wb.e[i].chunks = ep.chunks;
      wb.e[i].block_begin = wblocks;
      wblocks += (int)ceil_div(ep.L, 256);
    }
    HIP_TRY(launch_ngram_weight(wb, wblocks, n, w_min, partial, canon, exposure, weights, s), "ngram_weight");
  }
  return ATTT_OK;
}
}  // namespace

// ------------------------------------------------------------------------------------------
// Attention-block backward
// ------------------------------------------------------------------------------------------
extern "C" attt_status attt_attention_bwd(const void* q, const void* k, const void* v, const void* dout,
                                          const int64_t* row_offsets, int32_t num_episodes, int64_t N,
                                          int32_t heads, int32_t kv_heads, int32_t head_dim, float scale,
                                          void* dq, void* dk, void* dv, float* lse, float* dsum, void* stream) {
  if (head_dim != 128) return fail(ATTT_EUNSUPPORTED, "attention: head_dim must be 128 (got %d)", head_dim);
  if (heads < 1 || kv_heads < 1 || heads % kv_heads != 0)
    return fail(ATTT_EINVAL, "attention: heads (%d) must be a positive multiple of kv_heads (%d)", heads, kv_heads);
  if (!(scale > 0.0f) || !std::isfinite(scale)) return fail(ATTT_EINVAL, "attention: scale must be finite and > 0");
  if (N < 0) return fail(ATTT_EINVAL, "attention: N must be >= 0");
  if (N * heads >= INT32_MAX) return fail(ATTT_EUNSUPPORTED, "attention: N x heads must be < 2^31");
  if (heads >= (1 << 16)) return fail(ATTT_EUNSUPPORTED, "attention: heads must be < 2^16 (got %d)", heads);
  if (num_episodes < 1) return fail(ATTT_EINVAL, "attention: num_episodes must be >= 1 (got %d)", num_episodes);
  int64_t single[2] = {0, N};
  const int64_t* off = row_offsets;
  if (!off) {
    if (num_episodes != 1) return fail(ATTT_EINVAL, "attention: row_offsets may be NULL only for one episode");
    off = single;
  }
  attt_status st = check_offsets("attention rows", off, num_episodes, INT32_MAX);
  if (st) return st;
  if (off[num_episodes] != N)
    return fail(ATTT_EINVAL, "attention: row_offsets[E] (%lld) != N (%lld)", (long long)off[num_episodes], (long long)N);
  if (N == 0) return ATTT_OK;
  const void* ptrs[] = {q, k, v, dout, dq, dk, dv, lse, dsum};
  for (const void* ptr : ptrs) {
    if (!ptr) return fail(ATTT_EINVAL, "attention: null pointer");
    if (!aligned16(ptr)) return fail(ATTT_EINVAL, "attention: device pointers must be 16-byte aligned");
  }
  AttnArgs a{};
  a.q = static_cast<const bf16_t*>(q);
  a.k = static_cast<const bf16_t*>(k);
  a.v = static_cast<const bf16_t*>(v);
  a.dout = static_cast<const bf16_t*>(dout);
  a.dq = static_cast<bf16_t*>(dq);
  a.dk = static_cast<bf16_t*>(dk);
  a.dv = static_cast<bf16_t*>(dv);
  a.lse = lse;
  a.dsum = dsum;
  a.N = (int32_t)N;
  a.heads = heads;
  a.kv_heads = kv_heads;
  a.scale = scale;
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int32_t e0 = 0; e0 < num_episodes; e0 += kEpBatch) {
    AttnBatch b{};
    b.count = std::min<int32_t>(kEpBatch, num_episodes - e0);
    for (int i = 0; i < b.count; ++i) {
      b.e[i].row0 = off[e0 + i];
      b.e[i].L = (int32_t)(off[e0 + i + 1] - off[e0 + i]);
      b.e[i].blocks = (int32_t)ceil_div(b.e[i].L, 64);
    }
    // workgroups per episode: blocks x heads (forward statistics, dQ) or x kv_heads (dK, dV)
    for (int kernel = 0; kernel < 3; ++kernel) {
      const int per = kernel == 1 ? kv_heads : heads;
      int wgs = 0;
      for (int i = 0; i < b.count; ++i) {
        b.e[i].wg_begin = wgs;
        wgs += b.e[i].blocks * per;
      }
      HIP_TRY(launch_attn(kernel, a, b, wgs, s), kernel == 0 ? "attn_fwd_stats" : kernel == 1 ? "attn_dkdv" : "attn_dq");
    }
  }
  return ATTT_OK;
}

// ------------------------------------------------------------------------------------------
// Update-text repetition (Eq. 6-7)
// ------------------------------------------------------------------------------------------
namespace {
constexpr int64_t kRepMaxTextWords = (int64_t)1 << 20;
constexpr int64_t kRepMaxRecords = (int64_t)1 << 26;

struct RepPlan {
  std::vector<RepEp> eps;  // wg_begin relative to the episode's launch batch is set at launch
  int64_t records = 0, pairs = 0;
  size_t total = 0;
};

attt_status rep_plan(const int64_t* toff, const int64_t* etx, int32_t E, RepPlan& P) {
  if (E < 1) return fail(ATTT_EINVAL, "repetition: num_episodes must be >= 1 (got %d)", E);
  if (!toff || !etx) return fail(ATTT_EINVAL, "repetition: offsets pointer is null");
  if (etx[0] != 0) return fail(ATTT_EINVAL, "repetition: episode_texts[0] must be 0");
  for (int32_t e = 0; e < E; ++e)
    if (etx[e + 1] <= etx[e]) return fail(ATTT_EINVAL, "repetition: episode %d has no text", e);
  const int64_t T = etx[E];
  if (T > INT32_MAX) return fail(ATTT_EUNSUPPORTED, "repetition: %lld texts (limit 2^31 - 1)", (long long)T);
  if (toff[0] != 0) return fail(ATTT_EINVAL, "repetition: text_offsets[0] must be 0");
  for (int64_t t = 0; t < T; ++t) {
    if (toff[t + 1] < toff[t]) return fail(ATTT_EINVAL, "repetition: text_offsets decrease at text %lld", (long long)t);
    if (toff[t + 1] - toff[t] > kRepMaxTextWords)
      return fail(ATTT_EUNSUPPORTED, "repetition: text %lld holds %lld words (limit 2^20)", (long long)t,
                  (long long)(toff[t + 1] - toff[t]));
  }
  if (toff[T] > INT32_MAX) return fail(ATTT_EUNSUPPORTED, "repetition: %lld words (limit 2^31 - 1)", (long long)toff[T]);
  for (int32_t e = 0; e < E; ++e) {
    RepEp ep{};
    ep.text0 = etx[e];
    ep.ntexts = (int32_t)(etx[e + 1] - etx[e]);
    ep.ep = e;
    const int64_t cand = etx[e + 1] - 1;
    int64_t longest = toff[cand + 1] - toff[cand];
    for (int64_t t = etx[e]; t < cand; ++t) longest = std::max(longest, toff[t + 1] - toff[t]);
    // a partition sees about kRepPartWords words of each text: its LDS sets stay below 1/4 full
    ep.parts = (int32_t)std::max<int64_t>(1, ceil_div(longest, kRepPartWords));
    ep.wg_global = P.records;
    ep.pair_base = P.pairs;
    P.records += (int64_t)(ep.ntexts - 1) * ep.parts;
    P.pairs += ep.ntexts - 1;
    P.eps.push_back(ep);
  }
  if (P.records > kRepMaxRecords)
    return fail(ATTT_EUNSUPPORTED, "repetition: %lld pairs x partitions (limit 2^26)", (long long)P.records);
  P.total = std::max<size_t>(align256((size_t)P.records * 16), 256);
  return ATTT_OK;
}
}  // namespace

extern "C" attt_status attt_repetition_workspace_size(const int64_t* text_offsets, const int64_t* episode_texts,
                                                      int32_t num_episodes, size_t* bytes) {
  if (!bytes) return fail(ATTT_EINVAL, "repetition: bytes is null");
  RepPlan P;
  attt_status st = rep_plan(text_offsets, episode_texts, num_episodes, P);
  if (st) return st;
  *bytes = P.total;
  return ATTT_OK;
}

extern "C" attt_status attt_update_repetition(const int32_t* words, const int64_t* text_offsets,
                                              const int64_t* text_offsets_dev, const int64_t* episode_texts,
                                              int32_t num_episodes, double tau, double* rho, double* nu,
                                              int32_t* skip, int32_t* best, int32_t* pair_counts,
                                              void* workspace, size_t workspace_bytes, void* stream) {
  RepPlan P;
  attt_status st = rep_plan(text_offsets, episode_texts, num_episodes, P);
  if (st) return st;
  if (!std::isfinite(tau)) return fail(ATTT_EINVAL, "repetition: tau must be finite");
  if (!rho || !nu || !skip || !best) return fail(ATTT_EINVAL, "repetition: null output pointer");
  if (!text_offsets_dev) return fail(ATTT_EINVAL, "repetition: text_offsets_dev is null");
  if (text_offsets[episode_texts[num_episodes]] > 0 && !words) return fail(ATTT_EINVAL, "repetition: words is null");
  if (workspace_bytes < P.total)
    return fail(ATTT_ENOSPACE, "repetition: workspace %zu bytes, need %zu", workspace_bytes, P.total);
  if (!workspace) return fail(ATTT_EINVAL, "repetition: workspace is null");
  if (!aligned256(workspace)) return fail(ATTT_EINVAL, "repetition: workspace must be 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* counts = static_cast<int32_t*>(workspace);
  for (size_t e0 = 0; e0 < P.eps.size(); e0 += kEpBatch) {
    RepBatch b{};
    b.count = (int32_t)std::min<size_t>(kEpBatch, P.eps.size() - e0);
    int wgs = 0;
    for (int i = 0; i < b.count; ++i) {
      b.e[i] = P.eps[e0 + i];
      b.e[i].wg_begin = wgs;
      wgs += (b.e[i].ntexts - 1) * b.e[i].parts;
    }
    HIP_TRY(launch_rep_count(b, wgs, words, text_offsets_dev, counts, s), "rep_count");
    HIP_TRY(launch_rep_reduce(b, counts, tau, rho, nu, skip, best, pair_counts, s), "rep_reduce");
  }
  return ATTT_OK;
}

// ------------------------------------------------------------------------------------------
// Persistent n-gram sets
// ------------------------------------------------------------------------------------------
namespace {
constexpr int64_t kSetMaxCapacity = (int64_t)1 << 30;

// Table slots: a power of two at least twice the capacity (load factor at most 1/2).
int64_t set_slots(int64_t capacity) {
  int64_t S = 64;
  while (S < 2 * capacity) S *= 2;
  return S;
}

attt_status set_validate(void* const* sets, int32_t num_sets, int64_t capacity, int32_t n) {
  if (num_sets < 1) return fail(ATTT_EINVAL, "ngram_set: num_sets must be >= 1 (got %d)", num_sets);
  if (n < 1 || n > ATTT_NGRAM_MAX_N)
    return fail(ATTT_EINVAL, "ngram_set: n must be in [1, %d] (got %d)", ATTT_NGRAM_MAX_N, n);
  if (capacity < 1 || capacity > kSetMaxCapacity)
    return fail(ATTT_EINVAL, "ngram_set: capacity must be in [1, 2^30] (got %lld)", (long long)capacity);
  if (!sets) return fail(ATTT_EINVAL, "ngram_set: sets is null");
  for (int32_t e = 0; e < num_sets; ++e) {
    if (!sets[e]) return fail(ATTT_EINVAL, "ngram_set: set %d is null", e);
    if (!aligned256(sets[e])) return fail(ATTT_EINVAL, "ngram_set: set %d must be 256-byte aligned", e);
  }
  return ATTT_OK;
}

// Episode batches of the append and weights calls: ceil(L/256) blocks per set.
template <class Fn>
attt_status set_batches(void* const* sets, const int64_t* toff, int32_t E, Fn&& fn) {
  for (int32_t e0 = 0; e0 < E; e0 += kEpBatch) {
    NgramSetBatch b{};
    b.count = std::min<int32_t>(kEpBatch, E - e0);
    int blocks = 0;
    for (int i = 0; i < b.count; ++i) {
      const int64_t L = toff[e0 + i + 1] - toff[e0 + i];
      b.j[i].set = sets[e0 + i];
      b.j[i].tok_base = toff[e0 + i];
      b.j[i].L = (int32_t)L;
      b.j[i].block_begin = blocks;
      blocks += (int)ceil_div(L, 256);
    }
    attt_status st = fn(b, blocks);
    if (st) return st;
  }
  return ATTT_OK;
}
}  // namespace

extern "C" attt_status attt_ngram_set_size(int64_t capacity, int32_t n, size_t* bytes) {
  if (n < 1 || n > ATTT_NGRAM_MAX_N)
    return fail(ATTT_EINVAL, "ngram_set: n must be in [1, %d] (got %d)", ATTT_NGRAM_MAX_N, n);
  if (capacity < 1 || capacity > kSetMaxCapacity)
    return fail(ATTT_EINVAL, "ngram_set: capacity must be in [1, 2^30] (got %lld)", (long long)capacity);
  if (!bytes) return fail(ATTT_EINVAL, "ngram_set: bytes is null");
  *bytes = ngram_set_bytes(set_slots(capacity), n);
  return ATTT_OK;
}

extern "C" attt_status attt_ngram_set_init(void* const* sets, int32_t num_sets, int64_t capacity, int32_t n,
                                           size_t set_bytes, void* stream) {
  attt_status st = set_validate(sets, num_sets, capacity, n);
  if (st) return st;
  const int64_t S = set_slots(capacity);
  if (set_bytes < ngram_set_bytes(S, n))
    return fail(ATTT_ENOSPACE, "ngram_set: %zu bytes per set, need %zu", set_bytes, ngram_set_bytes(S, n));
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int32_t e0 = 0; e0 < num_sets; e0 += kEpBatch) {
    NgramSetBatch b{};
    b.count = std::min<int32_t>(kEpBatch, num_sets - e0);
    for (int i = 0; i < b.count; ++i) b.j[i].set = sets[e0 + i];
    HIP_TRY(launch_ngram_set_init(b, S, n, s), "ngram_set_init");
  }
  return ATTT_OK;
}

extern "C" attt_status attt_ngram_set_append(void* const* sets, const int32_t* tokens,
                                             const int64_t* token_offsets, int32_t num_sets,
                                             int64_t capacity, int32_t n, void* stream) {
  attt_status st = set_validate(sets, num_sets, capacity, n);
  if (st) return st;
  st = check_offsets("ngram_set tokens", token_offsets, num_sets, INT32_MAX);
  if (st) return st;
  if (token_offsets[num_sets] > 0 && !tokens) return fail(ATTT_EINVAL, "ngram_set: tokens is null");
  if (token_offsets[num_sets] >= ((int64_t)1 << 31))
    return fail(ATTT_EUNSUPPORTED, "ngram_set: more than 2^31-1 tokens in one call");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t S = set_slots(capacity);
  return set_batches(sets, token_offsets, num_sets, [&](const NgramSetBatch& b, int blocks) -> attt_status {
    HIP_TRY(launch_ngram_set_append(b, blocks, tokens, S, capacity, n, s), "ngram_set_append");
    return ATTT_OK;
  });
}

extern "C" attt_status attt_ngram_set_weights(void* const* sets, const int32_t* tokens,
                                              const int64_t* token_offsets, int32_t num_sets,
                                              int64_t capacity, int32_t n, float w_min,
                                              uint32_t* exposure, float* weights, void* stream) {
  attt_status st = set_validate(sets, num_sets, capacity, n);
  if (st) return st;
  if (!(w_min >= 0x1p-20f && w_min <= 1.0f))
    return fail(ATTT_EINVAL, "ngram_set: w_min must be in [2^-20, 1] (got %g)", (double)w_min);
  st = check_offsets("ngram_set tokens", token_offsets, num_sets, INT32_MAX);
  if (st) return st;
  const int64_t T = token_offsets[num_sets];
  if (T >= ((int64_t)1 << 31)) return fail(ATTT_EUNSUPPORTED, "ngram_set: more than 2^31-1 tokens in one call");
  if (T > 0 && !tokens) return fail(ATTT_EINVAL, "ngram_set: tokens is null");
  if (T > 0 && !weights) return fail(ATTT_EINVAL, "ngram_set: weights is null");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t S = set_slots(capacity);
  return set_batches(sets, token_offsets, num_sets, [&](const NgramSetBatch& b, int blocks) -> attt_status {
    HIP_TRY(launch_ngram_set_weights(b, blocks, tokens, S, n, w_min, exposure, weights, s), "ngram_set_weights");
    return ATTT_OK;
  });
}

// ------------------------------------------------------------------------------------------
// Weighted cross-entropy
// ------------------------------------------------------------------------------------------
namespace {

// float32 backward (three VALU GEMMs) blocking: rows per block and vocab columns per staged dZ
// chunk. The bf16 backward stages nothing of that shape (ce_fused.hip).
constexpr int64_t kCeRowBlock = 8192;
constexpr int64_t kCeVocabChunk = 131072;

struct CePlan {
  CeGemmShape fwd{64, 64};
  int64_t n_vb = 0, nv = 0, R = 0, Vc = 0, Vp = 0;
  int slices = 0, consumers = 0, passes = 0, ksplit = 1, slots = 0, items_max = 0, sync_ints = 0;
  size_t off_part = 0, off_label = 0, off_lse = 0, off_coef = 0, off_rowloss = 0;
  size_t off_flag = 0, off_sync = 0, off_sync2 = 0, off_ring = 0, off_split = 0;
  size_t off_wt = 0, off_dz = 0, total = 0;
};

CeGemmShape mfma_shape(int64_t rows, int64_t cols) {
  const int64_t big = ceil_div(rows, 256) * ceil_div(cols, 256);
  return big >= 512 ? CeGemmShape{256, 256} : CeGemmShape{128, 128};
}

// Largest V of the bf16 backward: the dH GEMM reads 256 rows of the transposed head [d, Vp]
// through one buffer descriptor of 1 GiB, so 256 * Vp * 2 bytes must stay below 2^30.
constexpr int64_t kCeMaxVBf16Grad = ((int64_t)1 << 21) - 256;

attt_status ce_validate(int64_t N, int64_t d, int64_t V, int32_t dtype, bool grad) {
  if (dtype != ATTT_F32 && dtype != ATTT_BF16) return fail(ATTT_EINVAL, "ce: unknown dtype %d", dtype);
  if (N < 0) return fail(ATTT_EINVAL, "ce: N must be >= 0 (got %lld)", (long long)N);
  if (d < 1 || d % 8 != 0) return fail(ATTT_EINVAL, "ce: d must be a positive multiple of 8 (got %lld)", (long long)d);
  if (V < 1) return fail(ATTT_EINVAL, "ce: V must be >= 1 (got %lld)", (long long)V);
  if (N >= ((int64_t)1 << 31) || V >= ((int64_t)1 << 31) || d >= ((int64_t)1 << 20))
    return fail(ATTT_EUNSUPPORTED, "ce: dimensions beyond this build's limits");
  if (dtype == ATTT_BF16 && grad && V > kCeMaxVBf16Grad)
    return fail(ATTT_EUNSUPPORTED, "ce: the bf16 backward supports V <= %lld (got %lld)",
                (long long)kCeMaxVBf16Grad, (long long)V);
  return ATTT_OK;
}

CePlan ce_plan(int64_t N, int64_t d, int64_t V, int32_t dtype, bool grad, bool have_head_t) {
  CePlan P;
  if (dtype == ATTT_BF16) {
    P.fwd = mfma_shape(N, V);
    P.Vp = round_up(V, 256);
  } else {
    P.Vc = std::min<int64_t>(round_up(V, 64), kCeVocabChunk);
    P.R = std::min<int64_t>(std::max<int64_t>(N, 1), kCeRowBlock);
    P.Vp = V;
  }
  P.n_vb = ceil_div(V, P.fwd.bn);
  P.nv = ceil_div(V, 256);
  // The (max, sum) partials of the forward and the per-(row, vocab tile) sums of the fused
  // backward share one region: the sums are consumed before the exact path writes partials.
  const size_t part = std::max((size_t)N * P.n_vb * 8, dtype == ATTT_BF16 ? (size_t)N * P.nv * 4 : 0);
  size_t o = 0;
  P.off_part = o;    o += align256(part);
  P.off_label = o;   o += align256((size_t)N * 4);
  P.off_lse = o;     o += align256((size_t)N * 4);
  P.off_coef = o;    o += align256((size_t)N * 4);
  P.off_rowloss = o; o += align256((size_t)N * 4);
  if (grad && N > 0) {
    if (dtype == ATTT_BF16) {
      // fused backward: one consumer per 256-column slice of d (at most 24 of a team of
      // kCeTeam; more slices take several passes), the rest produce; the ring gives every
      // producer two slots plus slack
      P.slices = (int)ceil_div(d, 256);
      // A producer's item costs slices times a consumer's share of it. With fewer than 16 slices,
      // F = 16 / slices consumers per slice split the vocabulary tiles between them, so that
      // producers and consumers stay near 16 each; their sums meet in a fixed order.
      P.ksplit = P.slices < 16 ? (int)std::max<int64_t>(1, std::min<int64_t>(16 / P.slices, P.nv)) : 1;
      P.consumers = P.ksplit > 1 ? P.slices * P.ksplit : std::min(P.slices, 24);
      P.passes = (int)ceil_div(P.slices, P.consumers);
      P.slots = 2 * (kCeTeam - P.consumers) + 4;
      // items of the busiest team: its row tiles (one in 8) x passes x vocabulary tiles
      P.items_max = (int)round_up(ceil_div(ceil_div(N, 256), 8) * P.passes * P.nv, 4);
      P.sync_ints = ce_fused_sync_ints(P.slots, P.items_max);
      P.off_flag = o;  o += 256;
      P.off_sync = o;  o += align256((size_t)P.sync_ints * 4);
      P.off_sync2 = o; o += align256((size_t)P.sync_ints * 4);
      P.off_ring = o;  o += align256(ce_fused_ring_bytes(P.slots));
      if (P.ksplit > 1) {
        P.off_split = o;
        o += align256((size_t)8 * P.slices * (P.ksplit - 1) * 256 * 256 * sizeof(float));
      }
      if (!have_head_t) {
        P.off_wt = o;
        o += align256((size_t)d * P.Vp * 2);
      }
    } else {
      P.off_dz = o;
      o += align256((size_t)P.R * P.Vc * 4);
    }
  }
  P.total = std::max<size_t>(o, 256);
  return P;
}

// The fused backward runs one workgroup per CU in teams of kCeTeam per XCD: the 256-CU, 8-XCD
// layout of the MI355X, with cooperative launch. Cached per device.
attt_status ce_fused_device_ok() {
  static std::mutex mu;
  static int state[64] = {};  // 0 unknown, 1 ok, 2 not
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(ATTT_EUNSUPPORTED, "ce: device index %d", dev);
  std::lock_guard<std::mutex> lk(mu);
  if (state[dev] == 0) {
    int cus = 0, coop = 0;
    HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "hipDeviceGetAttribute");
    HIP_TRY(hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev), "hipDeviceGetAttribute");
    state[dev] = (cus == 8 * kCeTeam && coop) ? 1 : 2;
    if (state[dev] == 2)
      return fail(ATTT_EUNSUPPORTED, "ce: the bf16 backward needs %d CUs and cooperative launch (device has %d CUs%s)",
                  8 * kCeTeam, cus, coop ? "" : ", no cooperative launch");
  }
  if (state[dev] == 2) return fail(ATTT_EUNSUPPORTED, "ce: the bf16 backward needs %d CUs and cooperative launch",
                                   8 * kCeTeam);
  return ATTT_OK;
}

// bounds of the fused backward's waits (microseconds): label-referenced pass, exact pass
int64_t g_ce_wait_us[2] = {20000, 20000};

}  // namespace

extern "C" attt_status attt_ce_workspace_size(int64_t N, int64_t d, int64_t V, int32_t dtype,
                                              int32_t flags, size_t* bytes) {
  if (!bytes) return fail(ATTT_EINVAL, "ce: bytes is null");
  if (flags & ~(ATTT_CE_WANT_GRAD | ATTT_CE_HEAD_T)) return fail(ATTT_EINVAL, "ce: unknown flags 0x%x", flags);
  const bool grad = (flags & ATTT_CE_WANT_GRAD) != 0;
  attt_status st = ce_validate(N, d, V, dtype, grad);
  if (st) return st;
  *bytes = ce_plan(N, d, V, dtype, grad, (flags & ATTT_CE_HEAD_T) != 0).total;
  return ATTT_OK;
}

extern "C" attt_status attt_ce_head_t_size(int64_t d, int64_t V, size_t* bytes) {
  if (!bytes) return fail(ATTT_EINVAL, "ce_head_t: bytes is null");
  attt_status st = ce_validate(0, d, V, ATTT_BF16, true);
  if (st) return st;
  *bytes = (size_t)d * round_up(V, 256) * 2;
  return ATTT_OK;
}

extern "C" attt_status attt_ce_head_transpose(const void* lm_head, int64_t d, int64_t V, void* lm_head_t,
                                              size_t lm_head_t_bytes, void* stream) {
  attt_status st = ce_validate(0, d, V, ATTT_BF16, true);
  if (st) return st;
  if (!lm_head || !lm_head_t) return fail(ATTT_EINVAL, "ce_head_t: null pointer");
  if (!aligned16(lm_head) || !aligned16(lm_head_t))
    return fail(ATTT_EINVAL, "ce_head_t: lm_head and lm_head_t must be 16-byte aligned");
  const int64_t Vp = round_up(V, 256);
  if (lm_head_t_bytes < (size_t)d * Vp * 2)
    return fail(ATTT_ENOSPACE, "ce_head_t: %zu bytes, need %zu", lm_head_t_bytes, (size_t)d * Vp * 2);
  HIP_TRY(launch_ce_head_transpose(lm_head, (int)V, (int)d, (int)Vp, lm_head_t, static_cast<hipStream_t>(stream)),
          "ce_head_transpose");
  return ATTT_OK;
}

extern "C" attt_status attt_weighted_ce_fwd_bwd(const void* hidden, const void* lm_head,
                                                const int32_t* labels, const float* weights,
                                                const int64_t* row_offsets, int32_t num_episodes,
                                                int64_t N, int64_t d, int64_t V, int32_t dtype,
                                                float* loss, float* lse, void* grad_hidden,
                                                void* workspace, size_t workspace_bytes,
                                                void* stream) {
  return attt_weighted_ce_fwd_bwd_ex(hidden, lm_head, nullptr, labels, weights, row_offsets, num_episodes, N,
                                     d, V, dtype, loss, lse, grad_hidden, workspace, workspace_bytes, stream);
}

extern "C" attt_status attt_weighted_ce_fwd_bwd_ex(const void* hidden, const void* lm_head,
                                                   const void* lm_head_t, const int32_t* labels,
                                                   const float* weights, const int64_t* row_offsets,
                                                   int32_t num_episodes, int64_t N, int64_t d, int64_t V,
                                                   int32_t dtype, float* loss, float* lse, void* grad_hidden,
                                                   void* workspace, size_t workspace_bytes, void* stream) {
  attt_status st = ce_validate(N, d, V, dtype, grad_hidden != nullptr);
  if (st) return st;
  if (lm_head_t && (dtype != ATTT_BF16 || !grad_hidden))
    return fail(ATTT_EINVAL, "ce: lm_head_t applies to the bf16 backward only");
  if (lm_head_t && !aligned16(lm_head_t)) return fail(ATTT_EINVAL, "ce: lm_head_t must be 16-byte aligned");
  if (num_episodes < 1) return fail(ATTT_EINVAL, "ce: num_episodes must be >= 1 (got %d)", num_episodes);
  int64_t single[2] = {0, N};
  const int64_t* off = row_offsets;
  if (!off) {
    if (num_episodes != 1) return fail(ATTT_EINVAL, "ce: row_offsets may be NULL only for one episode");
    off = single;
  }
  st = check_offsets("ce rows", off, num_episodes, INT32_MAX);
  if (st) return st;
  if (off[num_episodes] != N) return fail(ATTT_EINVAL, "ce: row_offsets[E] (%lld) != N (%lld)",
                                          (long long)off[num_episodes], (long long)N);
  if (!loss) return fail(ATTT_EINVAL, "ce: loss is null");
  if (N > 0) {
    if (!hidden || !lm_head || !labels || !weights) return fail(ATTT_EINVAL, "ce: null input pointer");
    if (!aligned16(hidden) || !aligned16(lm_head) || (grad_hidden && !aligned16(grad_hidden)))
      return fail(ATTT_EINVAL, "ce: hidden, lm_head and grad_hidden must be 16-byte aligned");
  }
  const bool grad = grad_hidden != nullptr;
  CePlan P = ce_plan(N, d, V, dtype, grad, lm_head_t != nullptr);
  if (workspace_bytes < P.total)
    return fail(ATTT_ENOSPACE, "ce: workspace %zu bytes, need %zu", workspace_bytes, P.total);
  if (!workspace) return fail(ATTT_EINVAL, "ce: workspace is null");
  if (!aligned256(workspace)) return fail(ATTT_EINVAL, "ce: workspace must be 256-byte aligned");

  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  float2* part = reinterpret_cast<float2*>(ws + P.off_part);
  float* label_logit = reinterpret_cast<float*>(ws + P.off_label);
  float* lse_buf = lse ? lse : reinterpret_cast<float*>(ws + P.off_lse);
  float* coef = reinterpret_cast<float*>(ws + P.off_coef);
  float* rowloss = reinterpret_cast<float*>(ws + P.off_rowloss);
  const int E = num_episodes;
  if (N == 0) {
    // every episode is empty: loss 0
    for (int e0 = 0; e0 < E; e0 += kEpBatch) {
      CeEpBatch b{};
      b.count = std::min(kEpBatch, E - e0);
      b.first = e0;
      for (int i = 0; i < b.count; ++i) b.e[i].row0 = 0;
      HIP_TRY(launch_ce_loss(b, rowloss, loss, nullptr, s), "ce_loss");
    }
    return ATTT_OK;
  }
  auto batches = [&](int rows_per_block, auto&& fn) -> attt_status {
    for (int e0 = 0; e0 < E; e0 += kEpBatch) {
      CeEpBatch b{};
      b.count = std::min(kEpBatch, E - e0);
      b.first = e0;
      int blocks = 0;
      for (int i = 0; i < b.count; ++i) {
        b.e[i].row0 = off[e0 + i];
        b.e[i].L = (int32_t)(off[e0 + i + 1] - off[e0 + i]);
        b.e[i].block_begin = blocks;
        blocks += (int)ceil_div(b.e[i].L, rows_per_block);
      }
      attt_status st2 = fn(b, blocks);
      if (st2) return st2;
    }
    return ATTT_OK;
  };
  const void* wt = !(grad && dtype == ATTT_BF16) ? nullptr : lm_head_t ? lm_head_t : ws + P.off_wt;
  // The forward (both dtypes; also the exact path of the bf16 backward, gated on `gate`):
  // (max, sum exp) partials -> lse, coef, w CE -> loss.
  auto forward = [&](const int* gate) -> attt_status {
    HIP_TRY(launch_ce_fwd(dtype, P.fwd, hidden, lm_head, labels, (int)N, (int)d, (int)V, part,
                          (int)P.n_vb, label_logit, gate, s),
            "ce_fwd_lse");
    return batches(4, [&](const CeEpBatch& b, int blocks) -> attt_status {
      HIP_TRY(launch_ce_row_reduce(b, blocks, part, (int)P.n_vb, label_logit, weights, lse_buf, coef,
                                   rowloss, gate, s),
              "ce_row_reduce");
      HIP_TRY(launch_ce_loss(b, rowloss, loss, gate, s), "ce_loss");
      return ATTT_OK;
    });
  };

  if (dtype == ATTT_F32) {
    // float32: three VALU GEMMs, dZ = coef (softmax - onehot) staged per (row block, vocab chunk)
    st = forward(nullptr);
    if (st || !grad) return st;
    float* dz = reinterpret_cast<float*>(ws + P.off_dz);
    for (int64_t r0 = 0; r0 < N; r0 += P.R) {
      const int64_t R = std::min(P.R, N - r0);
      for (int64_t c0 = 0; c0 < V; c0 += P.Vc) {
        const int64_t width = std::min(P.Vc, V - c0);
        HIP_TRY(launch_ce_bwd_dz(static_cast<const float*>(hidden), static_cast<const float*>(lm_head), labels,
                                 lse_buf, coef, (int)r0, (int)R, (int)d, (int)c0, (int)width, (int)V, dz, (int)P.Vc,
                                 s),
                "ce_bwd_dz");
        HIP_TRY(launch_ce_bwd_dh(dz, (int)P.Vc, static_cast<const float*>(lm_head), (int)r0, (int)R, (int)d, (int)c0,
                                 (int)round_up(width, 16), (int)V, static_cast<float*>(grad_hidden), c0 == 0, s),
                "ce_bwd_dh");
      }
    }
    return ATTT_OK;
  }

  HIP_TRY(launch_ce_label(hidden, lm_head, labels, (int)N, (int)d, (int)V, label_logit,
                          grad ? reinterpret_cast<int*>(ws + P.off_flag) : nullptr, s),
          "ce_label_logit");
  if (!grad) return forward(nullptr);

  // bf16 forward + backward: the fused label-referenced pass (ce_fused.hip), lse and the loss
  // from its per-tile sums, then the exact pass, which runs only if the guard flag was raised
  // (a label-referenced sum could overflow, or the fused pass aborted).
  st = ce_fused_device_ok();
  if (st) return st;
  int* flag = reinterpret_cast<int*>(ws + P.off_flag);
  int* sync = reinterpret_cast<int*>(ws + P.off_sync);
  int* sync2 = reinterpret_cast<int*>(ws + P.off_sync2);
  float* sig_part = reinterpret_cast<float*>(ws + P.off_part);
  st = batches(256, [&](const CeEpBatch& b, int blocks) -> attt_status {
    HIP_TRY(launch_ce_coef(b, blocks, weights, coef, s), "ce_coef");
    return ATTT_OK;
  });
  if (st) return st;
  if (!lm_head_t)
    HIP_TRY(launch_ce_head_transpose(lm_head, (int)V, (int)d, (int)P.Vp, ws + P.off_wt, s), "ce_head_transpose");
  // both sync areas are adjacent: one clear
  HIP_TRY(launch_ce_sync_clear(sync, (int)((P.off_sync2 - P.off_sync) / 4 + P.sync_ints), s), "ce_sync_clear");
  CeFusedArgs fa{};
  fa.h = static_cast<const bf16_t*>(hidden);
  fa.W = static_cast<const bf16_t*>(lm_head);
  fa.WT = static_cast<const bf16_t*>(wt);
  fa.labels = labels;
  fa.label_logit = label_logit;
  fa.lse = lse_buf;
  fa.coef = coef;
  fa.sig_part = sig_part;
  fa.grad = static_cast<bf16_t*>(grad_hidden);
  fa.ring = ws + P.off_ring;
  fa.sync = sync;
  fa.gate = flag;
  fa.limit = (uint64_t)g_ce_wait_us[0] * 100;
  fa.N = (int)N;
  fa.d = (int)d;
  fa.V = (int)V;
  fa.Vp = (int)P.Vp;
  fa.nv = (int)P.nv;
  fa.row_tiles = (int)ceil_div(N, 256);
  fa.slices = P.slices;
  fa.consumers = P.consumers;
  fa.passes = P.passes;
  fa.ksplit = P.ksplit;
  fa.partial = P.ksplit > 1 ? reinterpret_cast<float*>(ws + P.off_split) : nullptr;
  fa.slots = P.slots;
  fa.items_max = P.items_max;
  HIP_TRY(launch_ce_fused(true, fa, s), "ce_fused_bwd");
  HIP_TRY(launch_ce_row_final(0, (int)N, sig_part, (int)P.nv, label_logit, weights, coef, lse_buf, rowloss, nullptr,
                              nullptr, s),
          "ce_row_final");
  st = batches(4, [&](const CeEpBatch& b, int) -> attt_status {
    HIP_TRY(launch_ce_loss(b, rowloss, loss, nullptr, s), "ce_loss");
    return ATTT_OK;
  });
  if (st) return st;
  HIP_TRY(launch_ce_fused_status(sync, flag, s), "ce_fused_status");
  // exact path: forward lse, then the fused pass on coef (exp(z - lse) - onehot)
  st = forward(flag);
  if (st) return st;
  fa.sync = sync2;
  fa.limit = (uint64_t)g_ce_wait_us[1] * 100;
  HIP_TRY(launch_ce_fused(false, fa, s), "ce_fused_bwd (exact)");
  HIP_TRY(launch_ce_fused_nan(sync2, loss, E, lse_buf, (int)N, grad_hidden, N * d, s), "ce_fused_nan");
  return ATTT_OK;
}

extern "C" attt_status attt_ce_set_wait_limit(int64_t label_us, int64_t exact_us) {
  if (label_us < 0 || exact_us < 0 || label_us > ((int64_t)1 << 40) || exact_us > ((int64_t)1 << 40))
    return fail(ATTT_EINVAL, "ce_set_wait_limit: limits must be in [0, 2^40] microseconds");
  g_ce_wait_us[0] = label_us;
  g_ce_wait_us[1] = exact_us;
  return ATTT_OK;
}

// ------------------------------------------------------------------------------------------
// LoRA gradients
// ------------------------------------------------------------------------------------------
namespace {

struct LoraProb {
  int64_t bt_off, ut_off, dut_off, pa_off, pb_off;
  int32_t rp, rows_pad, splits;
};

struct LoraPlan {
  std::vector<LoraProb> prob;           // per problem (entries of problems with rows > 0 used)
  std::vector<std::vector<int>> chunks;  // problems sharing x, d_in and rows; <= 4 rank tiles each
  size_t total = 0;
};

attt_status lora_validate(const attt_lora_problem* p, int32_t count, int32_t dtype) {
  if (dtype != ATTT_F32 && dtype != ATTT_BF16) return fail(ATTT_EINVAL, "lora: unknown dtype %d", dtype);
  if (count < 0) return fail(ATTT_EINVAL, "lora: count must be >= 0");
  if (count > 0 && !p) return fail(ATTT_EINVAL, "lora: problems is null");
  for (int32_t i = 0; i < count; ++i) {
    const attt_lora_problem& q = p[i];
    if (q.rank < 1 || q.rank > ATTT_LORA_MAX_RANK)
      return fail(ATTT_EINVAL, "lora[%d]: rank must be in [1, %d] (got %d)", i, ATTT_LORA_MAX_RANK, q.rank);
    if (q.rows < 0 || q.d_in < 1 || q.d_out < 1 || q.d_in % 8 || q.d_out % 8)
      return fail(ATTT_EINVAL, "lora[%d]: need rows >= 0 and d_in, d_out positive multiples of 8", i);
    // pass 2 addresses a rank tile's [2][16, rows_pad] bf16 operand through one 32-bit range
    if (q.rows >= ((int64_t)1 << 24) || q.d_in >= ((int64_t)1 << 20) || q.d_out >= ((int64_t)1 << 20))
      return fail(ATTT_EUNSUPPORTED, "lora[%d]: dimensions beyond this build's limits (rows < 2^24, "
                  "d_in and d_out < 2^20)", i);
    if (!std::isfinite(q.scale)) return fail(ATTT_EINVAL, "lora[%d]: scale is not finite", i);
    if (!q.dA || !q.dB) return fail(ATTT_EINVAL, "lora[%d]: dA / dB is null", i);
    if (q.rows > 0 && (!q.x || !q.dy || !q.A || !q.B)) return fail(ATTT_EINVAL, "lora[%d]: null input", i);
    if (q.rows > 0 && (!aligned16(q.x) || !aligned16(q.dy) || !aligned16(q.A)))
      return fail(ATTT_EINVAL, "lora[%d]: x, dy and A must be 16-byte aligned", i);
  }
  return ATTT_OK;
}

LoraPlan lora_plan(const attt_lora_problem* p, int32_t count, int32_t dtype) {
  LoraPlan P;
  const size_t esz = dtype == ATTT_BF16 ? 2 : 4;
  const size_t lt_planes = dtype == ATTT_BF16 ? 2 : 1;
  P.prob.resize(count);
  // Problems reading the same x (same pointer, d_in and rows) share pass-1 and dA jobs.
  std::vector<int> tiles(count, 0);
  for (int32_t i = 0; i < count; ++i) {
    if (p[i].rows == 0) continue;
    tiles[i] = (int)ceil_div(p[i].rank, 16);
    bool placed = false;
    for (auto& ch : P.chunks) {
      const attt_lora_problem& f = p[ch[0]];
      int used = 0;
      for (int m : ch) used += tiles[m];
      if (f.x == p[i].x && f.d_in == p[i].d_in && f.rows == p[i].rows && used + tiles[i] <= kLoraMaxTiles) {
        ch.push_back(i);
        placed = true;
        break;
      }
    }
    if (!placed) P.chunks.push_back({i});
  }
  // Row splits of pass 2: about 512 rows (eight steps of 64) per workgroup, at most 16 splits;
  // shorter chains of dependent loads for more float32 partials.
  size_t o = 0;
  for (int32_t i = 0; i < count; ++i) {
    const attt_lora_problem& q = p[i];
    if (q.rows == 0) continue;
    LoraProb& Q = P.prob[i];
    Q.rp = tiles[i] * 16;
    Q.rows_pad = (int32_t)round_up(q.rows, kLoraRowTile);
    Q.splits = std::max(1, std::min(16, Q.rows_pad / 512));
    Q.bt_off = (int64_t)o;  o += align256((size_t)Q.rp * q.d_out * esz);
    // pass-1 results U^T and dU^T: float32, or for bf16 two planes (hi, lo) per rank tile
    Q.ut_off = (int64_t)o;  o += align256((size_t)Q.rp * Q.rows_pad * esz * lt_planes);
    Q.dut_off = (int64_t)o; o += align256((size_t)Q.rp * Q.rows_pad * esz * lt_planes);
    Q.pa_off = (int64_t)o;  o += align256((size_t)Q.rp * Q.splits * q.d_in * 4);
    Q.pb_off = (int64_t)o;  o += align256((size_t)Q.rp * Q.splits * q.d_out * 4);
  }
  P.total = std::max<size_t>(o, 256);
  return P;
}

// Launches `jobs` in batches of Batch::kCap; blocks(job) gives each job's workgroup count.
template <class Batch = void, class Job, class Blocks, class Launch>
attt_status lora_launch_all(const std::vector<Job>& jobs, Blocks blocks, Launch launch, const char* name) {
  using B = std::conditional_t<std::is_void_v<Batch>, LoraBatchOf<Job>, Batch>;
  for (size_t j0 = 0; j0 < jobs.size(); j0 += B::kCap) {
    B b{};
    b.count = (int32_t)std::min<size_t>(B::kCap, jobs.size() - j0);
    int total = 0;
    for (int i = 0; i < b.count; ++i) {
      b.j[i] = jobs[j0 + i];
      b.j[i].b_begin = total;
      total += blocks(b.j[i]);
    }
    HIP_TRY(launch(b, total), name);
  }
  return ATTT_OK;
}

}  // namespace

extern "C" attt_status attt_lora_workspace_size(const attt_lora_problem* problems, int32_t count,
                                                int32_t dtype, size_t* bytes) {
  if (!bytes) return fail(ATTT_EINVAL, "lora: bytes is null");
  attt_status st = lora_validate(problems, count, dtype);
  if (st) return st;
  *bytes = lora_plan(problems, count, dtype).total;
  return ATTT_OK;
}

extern "C" attt_status attt_lora_grad(const attt_lora_problem* problems, int32_t count, int32_t dtype,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  attt_status st = lora_validate(problems, count, dtype);
  if (st) return st;
  LoraPlan P = lora_plan(problems, count, dtype);
  if (workspace_bytes < P.total)
    return fail(ATTT_ENOSPACE, "lora: workspace %zu bytes, need %zu", workspace_bytes, P.total);
  if (!workspace) return fail(ATTT_EINVAL, "lora: workspace is null");
  if (!aligned256(workspace)) return fail(ATTT_EINVAL, "lora: workspace must be 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  const int64_t esz = dtype == ATTT_BF16 ? 2 : 4;
  const int64_t lt_tile = 16 * (dtype == ATTT_BF16 ? 2 : 1) * esz;  // bytes per row of rows_pad per tile

  std::vector<LoraBTJob> bt;
  std::vector<LoraP1Job> p1;
  std::vector<LoraP2Job> p2;
  std::vector<LoraRedJob> red;
  auto add_tile1 = [](LoraP1Job& J, const void* op, int valid, float scale, int64_t out_off) {
    LoraP1Tile& T = J.t[J.nt++];
    T.op = op;
    T.valid = valid;
    T.scale = scale;
    T.out_off = out_off;
  };
  auto add_tile2 = [](LoraP2Job& J, int64_t lt_off, int64_t part_off) {
    LoraP2Tile& T = J.t[J.nt++];
    T.lt_off = lt_off;
    T.part_off = part_off;
  };
  // x jobs (shared by a chunk's problems): U tiles in pass 1, dA tiles in pass 2
  for (const auto& ch : P.chunks) {
    const attt_lora_problem& f = problems[ch[0]];
    const LoraProb& F = P.prob[ch[0]];
    LoraP1Job J1{};
    J1.src = f.x;
    J1.rows = (int32_t)f.rows;
    J1.rows_pad = F.rows_pad;
    J1.kdim = (int32_t)f.d_in;
    LoraP2Job J2{};
    J2.src = f.x;
    J2.rows = (int32_t)f.rows;
    J2.rows_pad = F.rows_pad;
    J2.cols = (int32_t)f.d_in;
    J2.splits = F.splits;
    for (int i : ch) {
      const attt_lora_problem& q = problems[i];
      const LoraProb& Q = P.prob[i];
      for (int t = 0; t < Q.rp / 16; ++t) {
        add_tile1(J1, static_cast<const uint8_t*>(q.A) + (int64_t)16 * t * q.d_in * esz,
                  std::min(16, q.rank - 16 * t), q.scale, Q.ut_off + (int64_t)t * Q.rows_pad * lt_tile);
        add_tile2(J2, Q.dut_off + (int64_t)t * Q.rows_pad * lt_tile,
                  Q.pa_off + (int64_t)t * Q.splits * 16 * q.d_in * 4);
      }
    }
    p1.push_back(J1);
    p2.push_back(J2);
  }
  // dy jobs (one per problem): dU tiles in pass 1, dB tiles in pass 2; B^T; reduction
  for (int32_t i = 0; i < count; ++i) {
    const attt_lora_problem& q = problems[i];
    if (q.rows == 0) continue;
    const LoraProb& Q = P.prob[i];
    LoraBTJob JB{};
    JB.B = q.B;
    JB.bt_off = Q.bt_off;
    JB.rank = q.rank;
    JB.rp = Q.rp;
    JB.d_out = (int32_t)q.d_out;
    bt.push_back(JB);
    LoraP1Job J1{};
    J1.src = q.dy;
    J1.rows = (int32_t)q.rows;
    J1.rows_pad = Q.rows_pad;
    J1.kdim = (int32_t)q.d_out;
    LoraP2Job J2{};
    J2.src = q.dy;
    J2.rows = (int32_t)q.rows;
    J2.rows_pad = Q.rows_pad;
    J2.cols = (int32_t)q.d_out;
    J2.splits = Q.splits;
    for (int t = 0; t < Q.rp / 16; ++t) {
      add_tile1(J1, ws + Q.bt_off + (int64_t)16 * t * q.d_out * esz, 16, q.scale,
                Q.dut_off + (int64_t)t * Q.rows_pad * lt_tile);
      add_tile2(J2, Q.ut_off + (int64_t)t * Q.rows_pad * lt_tile,
                Q.pb_off + (int64_t)t * Q.splits * 16 * q.d_out * 4);
    }
    p1.push_back(J1);
    p2.push_back(J2);
    LoraRedJob JR{};
    JR.dA = q.dA;
    JR.dB = q.dB;
    JR.pa_off = Q.pa_off;
    JR.pb_off = Q.pb_off;
    JR.rank = q.rank;
    JR.d_in = (int32_t)q.d_in;
    JR.d_out = (int32_t)q.d_out;
    JR.sa = Q.splits;
    JR.sb = Q.splits;
    red.push_back(JR);
  }
  st = lora_launch_all(
      bt, [](const LoraBTJob& J) { return (int)ceil_div((int64_t)J.rp * J.d_out, 256); },
      [&](const LoraBTBatch& b, int n) { return launch_lora_bt(dtype, b, n, ws, s); }, "lora_bt");
  if (st) return st;
  // pass 1: jobs sorted by tile count, each launch specialised on its batch's largest count
  std::stable_sort(p1.begin(), p1.end(), [](const LoraP1Job& a, const LoraP1Job& b) { return a.nt > b.nt; });
  st = lora_launch_all(
      p1, [](const LoraP1Job& J) { return J.rows_pad / kLoraP1Rows; },
      [&](const LoraP1Batch& b, int n) { return launch_lora_pass1(dtype, b.j[0].nt, b, n, ws, s); }, "lora_u_du");
  if (st) return st;
  st = lora_launch_all(
      p2, [](const LoraP2Job& J) { return J.splits * (int)ceil_div(J.cols, kLoraColTile); },
      [&](const LoraP2Batch& b, int n) { return launch_lora_pass2(dtype, b, n, ws, s); }, "lora_dadb");
  if (st) return st;
  return lora_launch_all(
      red, [](const LoraRedJob& J) { return (int)ceil_div((int64_t)J.rank * J.d_in + (int64_t)J.d_out * J.rank, 256); },
      [&](const LoraRedBatch& b, int n) { return launch_lora_reduce(b, n, ws, s); }, "lora_reduce");
}

extern "C" attt_status attt_lora_sgd_step(const attt_lora_param* params, int32_t count, float lr,
                                          int32_t zero_grad, void* stream) {
  if (count < 0) return fail(ATTT_EINVAL, "lora_sgd: count must be >= 0");
  if (count > 0 && !params) return fail(ATTT_EINVAL, "lora_sgd: params is null");
  if (!std::isfinite(lr)) return fail(ATTT_EINVAL, "lora_sgd: lr is not finite");
  std::vector<LoraSgdJob> jobs;
  for (int32_t i = 0; i < count; ++i) {
    const attt_lora_param& q = params[i];
    if (q.n < 0) return fail(ATTT_EINVAL, "lora_sgd[%d]: n must be >= 0", i);
    if (q.n >= ((int64_t)1 << 31)) return fail(ATTT_EUNSUPPORTED, "lora_sgd[%d]: n beyond this build's limits", i);
    if (q.n == 0) continue;
    if (!q.param || !q.grad) return fail(ATTT_EINVAL, "lora_sgd[%d]: param / grad is null", i);
    if (reinterpret_cast<uintptr_t>(q.param) % 4 || reinterpret_cast<uintptr_t>(q.grad) % 4 ||
        reinterpret_cast<uintptr_t>(q.param_bf16) % 2)
      return fail(ATTT_EINVAL, "lora_sgd[%d]: misaligned array", i);
    LoraSgdJob J{};
    J.param = q.param;
    J.grad = q.grad;
    J.param_bf16 = static_cast<uint16_t*>(q.param_bf16);
    J.n = q.n;
    jobs.push_back(J);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  return lora_launch_all(
      jobs, [](const LoraSgdJob& J) { return (int)ceil_div(J.n, (int64_t)kLoraSgdPerBlock); },
      [&](const LoraSgdBatch& b, int n) { return launch_lora_sgd(b, n, lr, zero_grad, s); }, "lora_sgd");
}

// ------------------------------------------------------------------------------------------
// Serving: grouped multi-adapter forward, adapter swap
// ------------------------------------------------------------------------------------------
extern "C" attt_status attt_lora_forward(const attt_lora_fwd_problem* problems, int32_t count, void* stream) {
  if (count < 0) return fail(ATTT_EINVAL, "lora_forward: count must be >= 0");
  if (count > 0 && !problems) return fail(ATTT_EINVAL, "lora_forward: problems is null");
  for (int32_t i = 0; i < count; ++i) {
    const attt_lora_fwd_problem& q = problems[i];
    if (q.rank < 1 || q.rank > ATTT_LORA_MAX_RANK)
      return fail(ATTT_EINVAL, "lora_forward[%d]: rank must be in [1, %d] (got %d)", i, ATTT_LORA_MAX_RANK, q.rank);
    if (q.rows < 0 || q.d_in < 1 || q.d_out < 1 || q.d_in % 8 || q.d_out % 8)
      return fail(ATTT_EINVAL, "lora_forward[%d]: need rows >= 0 and d_in, d_out positive multiples of 8", i);
    // phase 1 addresses 16 rows of x, and a unit of A, through one 32-bit buffer range
    if (q.rows >= ((int64_t)1 << 24) || q.d_in >= ((int64_t)1 << 20) || q.d_out >= ((int64_t)1 << 20))
      return fail(ATTT_EUNSUPPORTED, "lora_forward[%d]: dimensions beyond this build's limits (rows < 2^24, "
                  "d_in and d_out < 2^20)", i);
    if (!std::isfinite(q.scale)) return fail(ATTT_EINVAL, "lora_forward[%d]: scale is not finite", i);
    if (q.rows > 0 && (!q.x || !q.y || !q.A || !q.B)) return fail(ATTT_EINVAL, "lora_forward[%d]: null array", i);
    if (q.rows > 0 && (!aligned16(q.x) || !aligned16(q.y) || !aligned16(q.A) || !aligned16(q.B)))
      return fail(ATTT_EINVAL, "lora_forward[%d]: x, y, A and B must be 16-byte aligned", i);
  }
  // jobs: problems reading the same x (pointer, d_in, rows), at most four 16-rank units each
  std::vector<std::vector<int>> groups;
  std::vector<int> units(count, 0);
  for (int32_t i = 0; i < count; ++i) {
    if (problems[i].rows == 0) continue;
    units[i] = (int)ceil_div(problems[i].rank, 16);
    bool placed = false;
    for (auto& gr : groups) {
      const attt_lora_fwd_problem& f = problems[gr[0]];
      int used = 0;
      for (int m : gr) used += units[m];
      if (f.x == problems[i].x && f.d_in == problems[i].d_in && f.rows == problems[i].rows &&
          used + units[i] <= kLoraMaxTiles) {
        gr.push_back(i);
        placed = true;
        break;
      }
    }
    if (!placed) groups.push_back({i});
  }
  // Jobs of at most 16 rows (decoding) run on 8-wave workgroups that split d_in eight ways;
  // larger jobs on 4-wave workgroups of 64 rows.
  std::vector<LoraFwdJob> jobs[2];  // [0] 4-wave, [1] 8-wave
  int64_t row_blocks = 0;
  int64_t max_dout = 8, max_dout_small = 8;
  for (const auto& gr : groups) {
    const attt_lora_fwd_problem& f = problems[gr[0]];
    const bool small = f.rows <= 16;
    LoraFwdJob J{};
    J.x = f.x;
    J.rows = (int32_t)f.rows;
    J.d_in = (int32_t)f.d_in;
    J.rb = small ? 16 : 64;
    J.kw = small ? 8 : 1;
    J.ncs = 1;
    for (int i : gr) {
      const attt_lora_fwd_problem& q = problems[i];
      LoraFwdOut& O = J.o[J.no++];
      O.B = q.B;
      O.y = q.y;
      O.d_out = (int32_t)q.d_out;
      O.rank = q.rank;
      O.u0 = 16 * J.nu;
      for (int t = 0; t < units[i]; ++t) {
        LoraFwdUnit& U = J.u[J.nu++];
        U.A = static_cast<const uint8_t*>(q.A) + (int64_t)16 * t * q.d_in * 2;
        U.valid = std::min(16, q.rank - 16 * t);
        U.scale = q.scale;
      }
      (small ? max_dout_small : max_dout) = std::max<int64_t>(small ? max_dout_small : max_dout, q.d_out);
    }
    if (!small) row_blocks += ceil_div(f.rows, J.rb);
    jobs[small ? 1 : 0].push_back(J);
  }
  // Few row blocks: split each block's columns over several workgroups, each recomputing x A^T
  // (x and A stay in the XCD's L2, the splits of a block running on one XCD), so that the
  // launch still fills the chip.
  int ncs = 1;
  if (row_blocks > 0 && row_blocks < 512)
    ncs = (int)std::min<int64_t>({16, ceil_div(1024, row_blocks), ceil_div(max_dout, 64)});
  ncs = std::max(ncs, 1);
  for (auto& J : jobs[0]) J.ncs = ncs;
  // decoding: every job's columns over up to 16 workgroups of at least 256 columns each
  const int ncs_small = (int)std::max<int64_t>(1, std::min<int64_t>(16, ceil_div(max_dout_small, 256)));
  for (auto& J : jobs[1]) J.ncs = ncs_small;
  hipStream_t s = static_cast<hipStream_t>(stream);
  for (int kind = 0; kind < 2; ++kind) {
    auto& js = jobs[kind];
    std::stable_sort(js.begin(), js.end(), [](const LoraFwdJob& a, const LoraFwdJob& b) { return a.nu > b.nu; });
    for (size_t j0 = 0; j0 < js.size(); j0 += kLoraFwdBatch) {
      LoraFwdBatch b{};
      b.count = (int32_t)std::min<size_t>(kLoraFwdBatch, js.size() - j0);
      int64_t total = 0;
      for (int i = 0; i < b.count; ++i) {
        b.j[i] = js[j0 + i];
        b.j[i].b_begin = (int32_t)total;
        total += ceil_div(b.j[i].rows, b.j[i].rb) * b.j[i].ncs;
      }
      if (total >= ((int64_t)1 << 31) - 8) return fail(ATTT_EUNSUPPORTED, "lora_forward: too many row blocks");
      b.total = (int32_t)total;
      HIP_TRY(launch_lora_fwd(b.j[0].nu, kind ? 8 : 4, b, s), "lora_fwd");
    }
  }
  return ATTT_OK;
}

extern "C" attt_status attt_lora_hot_swap(const attt_lora_swap_item* items, int32_t count, void* stream) {
  if (count < 0) return fail(ATTT_EINVAL, "lora_hot_swap: count must be >= 0");
  if (count > 0 && !items) return fail(ATTT_EINVAL, "lora_hot_swap: items is null");
  std::vector<LoraSwapJob> jobs;
  for (int32_t i = 0; i < count; ++i) {
    const attt_lora_swap_item& q = items[i];
    if (q.n < 0) return fail(ATTT_EINVAL, "lora_hot_swap[%d]: n must be >= 0", i);
    if (q.n >= ((int64_t)1 << 31)) return fail(ATTT_EUNSUPPORTED, "lora_hot_swap[%d]: n beyond this build's limits", i);
    if (q.n == 0) continue;
    if (!q.src || !q.dst) return fail(ATTT_EINVAL, "lora_hot_swap[%d]: src / dst is null", i);
    if (reinterpret_cast<uintptr_t>(q.src) % 4 || reinterpret_cast<uintptr_t>(q.dst) % 2)
      return fail(ATTT_EINVAL, "lora_hot_swap[%d]: misaligned array", i);
    LoraSwapJob J{};
    J.src = q.src;
    J.dst = static_cast<uint16_t*>(q.dst);
    J.n = q.n;
    J.vec = aligned16(q.src) && aligned16(q.dst);
    jobs.push_back(J);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  return lora_launch_all<LoraSwapBatch>(
      jobs, [](const LoraSwapJob& J) { return (int)ceil_div(J.n, (int64_t)kLoraSwapPerBlock); },
      [&](const LoraSwapBatch& b, int n) { return launch_lora_swap(b, n, s); }, "lora_swap");
}
