// n-gram exposure and token weights (Sec. 3.3, Eq. 8-9) on gfx950.
//
// Only the n-grams of the new update x_k matter for f, so the hash set is built over them
// (the small side: at most kQMax start positions per partition) and the history H^tok_k (the
// large side) is streamed once, coalesced, by many workgroups. Three kernels:
//
//   ngram_table_kernel   one workgroup per partition: inserts the partition's query n-grams
//                        into an LDS table of 4-entry buckets (hash tag | first query position
//                        with that n-gram) and writes, per query position, where its entry went
//                        (or that it repeats an earlier one) and its canonical position.
//   ngram_count_kernel   one workgroup per (partition, history chunk): rebuilds that table in LDS
//                        from the list (one store per distinct n-gram, no hashing), then every
//                        lane walks a run of 8 consecutive history positions with the tokens in
//                        registers and a rolling hash, looks each n-gram up with one 16-byte LDS
//                        read per bucket (a tag match is confirmed by comparing all n tokens),
//                        counts hits with LDS atomics, and writes the chunk's count of every
//                        canonical query n-gram (16 bits; a chunk has at most 65535 positions).
//   ngram_weight_kernel  per update token j: sums the chunk counts of the canonical n-grams of
//                        the starts that cover j in a fixed order, f(j) = their maximum, and
//                        w = max(w_min, 1 / (1 + f)) with a correctly rounded division.
//
// No global atomics and no hash table in global memory (the lists are per query position).
// Which position stands for a repeated n-gram depends on insertion order, but every position
// of the n-gram gets the same count, so f and w (integers, then one rounding) are
// bit-reproducible.
#include <mutex>
#include <utility>

#include "common.hpp"
#include "internal.hpp"

namespace attt {

// Scratch of the allocation-free entry point: the partial-count rows of the count kernel live
// in this file-scope array instead of a caller workspace. Host code never passes the array's
// name to a kernel (in host code it names a host-side stand-in); it passes the device address
// that hipGetSymbolAddress returns for the current device, looked up once per device.
static __device__ __align__(256) uint8_t scratch[kNgramScratchBytes];

hipError_t ngram_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

constexpr uint32_t kEmpty = 0xFFFFFFFFu;  // tag field of a real entry never has bit 31 set
constexpr uint32_t kNoSlot = 0xFFFFFFFFu; // list entry of a position that repeats an earlier n-gram
constexpr int kHalo = 16;                 // >= n - 1 extra query tokens after a partition
constexpr int kRun = 8;                   // consecutive history positions per lane

// Per-token 32-bit mix: full-rate 24-bit multiplies, a rotation folds the high product bits
// into the low ones. Only table placement depends on the hash: every tag match is verified
// token by token.
__device__ __forceinline__ uint32_t token_mix(int32_t t) {
  const uint32_t p = __umul24((uint32_t)t, 0x2F6B9Du) ^ (uint32_t)t;
  return p ^ __builtin_amdgcn_alignbit(p, p, 17);
}
__device__ __forceinline__ uint32_t rotl(uint32_t x, int r) { return __builtin_amdgcn_alignbit(x, x, (32 - r) & 31); }

// Cyclic-polynomial hash of n consecutive tokens: h = XOR_k rotl(g_k, n - 1 - k), g = token_mix.
// Moving the window by one token: h' = rotl(h, 1) ^ rotl(g_out, n) ^ g_in.
template <int N>
__device__ __forceinline__ uint32_t window_hash(const uint32_t* g) {
  uint32_t h = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) h = rotl(h, 1) ^ g[k];
  return h;
}

// Table placement of a hash: bucket from the low bits (folded), tag in bits 30..12 of the entry.
__device__ __forceinline__ uint32_t bucket_of(uint32_t h, uint32_t bmask) { return (h ^ (h >> 15)) & bmask; }
__device__ __forceinline__ uint32_t tag_of(uint32_t h) { return (h >> 1) & 0x7FFFF000u; }
constexpr uint32_t kTagMask = 0xFFFFF000u;

// All n comparisons from independent loads (query tokens in LDS against the window).
template <int N>
__device__ __forceinline__ bool ngram_equal(const int32_t* a, const int32_t* t) {
  bool eq = true;
#pragma unroll
  for (int i = 0; i < N; ++i) eq &= a[i] == t[i];
  return eq;
}

// One workgroup per partition of the batch.
template <int N>
__global__ __launch_bounds__(1024) void ngram_table_kernel(NgramPartBatch batch, const int32_t* __restrict__ tokens,
                                                           uint16_t* __restrict__ canon, uint2* __restrict__ list) {
  const NgramPart P = batch.p[blockIdx.x];
  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* tab = reinterpret_cast<uint32_t*>(smem);          // [slots], 4 per bucket
  int32_t* xs = reinterpret_cast<int32_t*>(tab + P.slots);    // [kQMax + kHalo]
  const int tid = threadIdx.x;
  const uint32_t bmask = (uint32_t)(P.slots >> 2) - 1u;
  const int32_t* x = tokens + P.tok_base + P.q0;
  for (int i = tid; i < P.slots; i += 1024) tab[i] = kEmpty;
  for (int i = tid; i < P.qn + N - 1; i += 1024) xs[i] = x[i];
  __syncthreads();
  // Slots of a bucket are claimed in order, so the occupied slots of every bucket form a prefix
  // and a bucket with a free slot ends every search. A repeated n-gram resolves to whichever of
  // its positions was inserted first.
  uint16_t* cn = canon + P.part_global * kQMax;
  uint2* ls = list + P.part_global * kQMax;
  for (int q = tid; q < P.qn; q += 1024) {
    uint32_t g[N];
#pragma unroll
    for (int k = 0; k < N; ++k) g[k] = token_mix(xs[q + k]);
    const uint32_t h = window_hash<N>(g);
    const uint32_t mine = tag_of(h) | (uint32_t)q;
    uint32_t b = bucket_of(h, bmask);
    int who = -1;
    uint32_t slot = kNoSlot;
    while (who < 0) {
#pragma unroll
      for (int sidx = 0; sidx < 4 && who < 0; ++sidx) {
        const uint32_t cur = atomicCAS(tab + b * 4 + sidx, kEmpty, mine);
        if (cur == kEmpty) {
          who = q;
          slot = b * 4 + sidx;
        } else if ((cur & kTagMask) == (mine & kTagMask) && ngram_equal<N>(xs + (cur & 0xFFFu), xs + q)) {
          who = (int)(cur & 0xFFFu);
        }
      }
      b = (b + 1u) & bmask;
    }
    cn[q] = (uint16_t)who;
    ls[q] = make_uint2(slot, mine);
  }
}

// Count-kernel table, rebuilt from the list: per bucket a signature word of four 8-bit tags
// (slot i in byte i; bit 7 set for an occupied slot, bits 6..0 from hash bits 31..25, i.e. the
// top of the table kernel's 19-bit tag) and, per slot, the query position (16 bits). One 4-byte
// read compares all four slots of a bucket.
__device__ __forceinline__ uint32_t sig_tag(uint32_t h) { return 0x80u | (h >> 25); }
// Bytes of x that are zero (bit 7 of each such byte set), exact: no borrow between bytes.
__device__ __forceinline__ uint32_t zero_bytes(uint32_t x) {
  return ~(((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x) & 0x80808080u;
}

// The general search: every matching slot of the bucket verified, then the following buckets
// while the current one is full. Returns the canonical query position, or -1.
template <int N>
__device__ __forceinline__ int probe_slow(const uint32_t* sig, const uint16_t* ent, const int32_t* xs,
                                                    uint32_t h, uint32_t bmask, const int32_t* t) {
  const uint32_t rep = __builtin_amdgcn_perm(0u, sig_tag(h), 0u);
  uint32_t b = bucket_of(h, bmask);
  while (true) {
    const uint32_t sg = sig[b];
    uint32_t z = zero_bytes(sg ^ rep);
    while (z) {
      const int i = __builtin_ctz(z) >> 3;
      const int q = ent[b * 4 + i];
      if (ngram_equal<N>(xs + q, t)) return q;
      z &= z - 1u;
    }
    if ((sg & 0x80808080u) != 0x80808080u) return -1;  // a free slot: the n-gram is not in the table
    b = (b + 1u) & bmask;
  }
}

template <int N>
__global__ __launch_bounds__(1024) void ngram_count_kernel(NgramPartBatch batch,
                                                           const int32_t* __restrict__ history,
                                                           const int32_t* __restrict__ tokens,
                                                           const uint2* __restrict__ list,
                                                           uint16_t* __restrict__ partial) {
  int pi = 0;
  while (pi + 1 < batch.count && batch.p[pi + 1].chunk_begin <= (int)blockIdx.x) ++pi;
  const NgramPart P = batch.p[pi];
  const int c = (int)blockIdx.x - P.chunk_begin;
  const int64_t per = (P.hist_ngrams + P.chunks - 1) / P.chunks;
  const int64_t i0 = (int64_t)c * per;
  const int64_t i1 = min((int64_t)P.hist_ngrams, i0 + per);

  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* sig = reinterpret_cast<uint32_t*>(smem);              // [slots / 4] signature words
  uint32_t* cnt = sig + P.slots / 4;                              // [kQMax / 2], 16-bit pairs
  int32_t* xs = reinterpret_cast<int32_t*>(cnt + kQMax / 2);      // [kQMax + kHalo]
  uint16_t* ent = reinterpret_cast<uint16_t*>(xs + kQMax + kHalo); // [slots] query positions
  const uint32_t bmask = (uint32_t)(P.slots >> 2) - 1u;
  const int tid = threadIdx.x;
  const int32_t* x = tokens + P.tok_base + P.q0;
  const uint2* ls = list + P.part_global * kQMax;

  // the table: every signature empty, then one tag byte and one position per distinct n-gram
  {
    u32x4* s4 = reinterpret_cast<u32x4*>(sig);
    for (int i = tid; i < P.slots / 16; i += 1024) s4[i] = u32x4{0u, 0u, 0u, 0u};
    for (int i = tid; i < kQMax / 2; i += 1024) cnt[i] = 0u;
    for (int i = tid; i < P.qn + N - 1; i += 1024) xs[i] = x[i];
  }
  __syncthreads();
  for (int q = tid; q < P.qn; q += 1024) {
    const uint2 e = ls[q];
    if (e.x != kNoSlot) {
      // entry bits 30..24 are hash bits 31..25 (tag_of), the signature's tag bits
      atomicOr(sig + (e.x >> 2), (0x80u | ((e.y >> 24) & 0x7Fu)) << ((e.x & 3u) * 8u));
      ent[e.x] = (uint16_t)(e.y & 0xFFFu);
    }
  }
  __syncthreads();

  // The chunk's history with its n-1 token halo is [i0, i1 + N - 1): the descriptor covers
  // exactly that range, so loads past its end return zero (and those positions are skipped).
  const __amdgpu_buffer_rsrc_t rh =
      buffer_rsrc(history + P.hist_base + i0, i1 > i0 ? (int)((i1 - i0 + N - 1) * 4) : 0);
  constexpr int W = kRun + N - 1;          // tokens of a lane's window
  constexpr int W4 = (W + 3) / 4;          // 16-byte loads
  // A lane's runs are kRun positions apart by 1024 * kRun; the next run's tokens are loaded while
  // this one is looked up (loads past the chunk's range return zero and are never used).
  u32x4 nxt[W4];
  auto fetch = [&](int64_t base) {
#pragma unroll
    for (int u = 0; u < W4; ++u)
      nxt[u] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rh, (uint32_t)(base - i0) * 4u + (uint32_t)u * 16u, 0, 0));
  };
  fetch(i0 + (int64_t)tid * kRun);
  for (int64_t g0 = i0; g0 < i1; g0 += 1024 * kRun) {
    const int64_t base = g0 + (int64_t)tid * kRun;
    int32_t t[W4 * 4];
#pragma unroll
    for (int u = 0; u < W4; ++u) {
      t[4 * u] = (int32_t)nxt[u][0];
      t[4 * u + 1] = (int32_t)nxt[u][1];
      t[4 * u + 2] = (int32_t)nxt[u][2];
      t[4 * u + 3] = (int32_t)nxt[u][3];
    }
    if (g0 + 1024 * kRun < i1) fetch(base + 1024 * kRun);
    if (base >= i1) continue;
    uint32_t g[W];
#pragma unroll
    for (int k = 0; k < W; ++k) g[k] = token_mix(t[k]);
    const int m = (int)min((int64_t)kRun, i1 - base);  // positions of this run inside the chunk
    uint32_t h = window_hash<N>(g);
#pragma unroll
    for (int p = 0; p < kRun; ++p) {
      if (p > 0) h = rotl(h, 1) ^ rotl(g[p - 1], N) ^ g[p + N - 1];
      // Fast path: one signature read; the lowest matching byte is verified. Anything else (a
      // failed verification with more matches, or no match in a full bucket) takes the slow
      // search. Lanes past the chunk's end do nothing.
      const uint32_t b = bucket_of(h, bmask);
      const uint32_t sg = sig[b];
      const uint32_t z = zero_bytes(sg ^ __builtin_amdgcn_perm(0u, sig_tag(h), 0u));
      int hit = -1;
      bool slow = false;
      if (p < m) {
        if (z) {
          const int q = ent[b * 4 + (__builtin_ctz(z) >> 3)];
          if (ngram_equal<N>(xs + q, t + p)) hit = q;
          else slow = (z & (z - 1u)) != 0u || (sg & 0x80808080u) == 0x80808080u;
        } else {
          slow = (sg & 0x80808080u) == 0x80808080u;
        }
      }
      if (slow) hit = probe_slow<N>(sig, ent, xs, h, bmask, t + p);
      if (hit >= 0) atomicAdd(cnt + (hit >> 1), 1u << ((hit & 1) * 16));
    }
  }
  __syncthreads();
  uint16_t* out = partial + (P.chunk_begin_global + c) * (int64_t)kQMax;
  for (int q = tid; q < (P.qn + 1) / 2; q += 1024) reinterpret_cast<uint32_t*>(out)[q] = cnt[q];
}

// 256 update tokens per block; the chunk counts of each n-gram start (through its canonical
// position) are summed by four groups of 256 threads (a quarter of the chunks each, several
// loads in flight per thread), then combined in LDS. Integer sums, so the order does not matter.
__global__ __launch_bounds__(1024) void ngram_weight_kernel(NgramEpBatch batch, int n, float w_min,
                                                            const uint16_t* __restrict__ partial,
                                                            const uint16_t* __restrict__ canon,
                                                            uint32_t* __restrict__ exposure,
                                                            float* __restrict__ weights) {
  int ei = 0;
  while (ei + 1 < batch.count && batch.e[ei + 1].block_begin <= (int)blockIdx.x) ++ei;
  const NgramEp E = batch.e[ei];
  const int j0 = ((int)blockIdx.x - E.block_begin) * 256;
  const int Q = E.L - n + 1;  // query start positions 0 .. Q-1
  __shared__ uint32_t cs[4][256 + kMaxN];
  const int grp = threadIdx.x >> 8, lt = threadIdx.x & 255;
  // counts of the starts s in [j0 - n + 1, j0 + 255] that exist
  const int s_lo = j0 - n + 1;
  for (int t = lt; t < 256 + n - 1; t += 256) {
    const int s = s_lo + t;
    uint32_t a0 = 0, a1 = 0, a2 = 0, a3 = 0;
    if (s >= 0 && s < Q && E.chunks > 0) {  // no history chunks: no canon rows, every count 0
      const int p = s / kQMax;
      const int r = canon[(E.part_base + p) * (int64_t)kQMax + (s - p * kQMax)];
      const uint16_t* col = partial + ((int64_t)E.chunk_base + (int64_t)p * E.chunks) * kQMax + r;
      int ch = grp;
#pragma unroll 4
      for (; ch + 12 < E.chunks; ch += 16) {
        a0 += col[(int64_t)ch * kQMax];
        a1 += col[(int64_t)(ch + 4) * kQMax];
        a2 += col[(int64_t)(ch + 8) * kQMax];
        a3 += col[(int64_t)(ch + 12) * kQMax];
      }
      for (; ch < E.chunks; ch += 4) a0 += col[(int64_t)ch * kQMax];
    }
    cs[grp][t] = (a0 + a1) + (a2 + a3);
  }
  __syncthreads();
  if (grp == 0)
    for (int t = lt; t < 256 + n - 1; t += 256) cs[0][t] = (cs[0][t] + cs[1][t]) + (cs[2][t] + cs[3][t]);
  __syncthreads();
  if (grp != 0) return;
  const int j = j0 + lt;
  if (j >= E.L) return;
  uint32_t f = 0;
  for (int i = 0; i < n; ++i) f = max(f, cs[0][lt + i]);  // starts j-n+1 .. j; absent ones hold 0
  const float w = fmaxf(w_min, __fdiv_rn(1.0f, 1.0f + (float)f));
  if (exposure) exposure[E.tok_base + j] = f;
  weights[E.tok_base + j] = w;
}

// ---------------------------------------------------------------------------------------
size_t ngram_count_lds(int slots, int n) {
  (void)n;
  return (size_t)slots + (size_t)kQMax * 2 + (size_t)(kQMax + kHalo) * 4 + (size_t)slots * 2;
}
static size_t ngram_table_lds(int slots) { return (size_t)slots * 4 + (size_t)(kQMax + kHalo) * 4; }

template <int N>
static hipError_t count_n(const NgramPartBatch& b, int total_blocks, size_t lds, const int32_t* history,
                          const int32_t* tokens, const uint2* list, uint16_t* partial, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)ngram_count_kernel<N>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL(ngram_count_kernel<N>, dim3(total_blocks), dim3(1024), lds, s, b, history, tokens, list,
                     partial);
  return hipGetLastError();
}

template <int N>
static hipError_t table_n(const NgramPartBatch& b, size_t lds, const int32_t* tokens, uint16_t* canon, uint2* list,
                          hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)ngram_table_kernel<N>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL(ngram_table_kernel<N>, dim3(b.count), dim3(1024), lds, s, b, tokens, canon, list);
  return hipGetLastError();
}

template <int... Ns>
static hipError_t count_dispatch(std::integer_sequence<int, Ns...>, int n, const NgramPartBatch& b,
                                 int total_blocks, size_t lds, const int32_t* history,
                                 const int32_t* tokens, const uint2* list, uint16_t* partial, hipStream_t s) {
  hipError_t e = hipErrorInvalidValue;
  ((n == Ns + 1 ? (e = count_n<Ns + 1>(b, total_blocks, lds, history, tokens, list, partial, s), 0) : 0), ...);
  return e;
}

template <int... Ns>
static hipError_t table_dispatch(std::integer_sequence<int, Ns...>, int n, const NgramPartBatch& b, size_t lds,
                                 const int32_t* tokens, uint16_t* canon, uint2* list, hipStream_t s) {
  hipError_t e = hipErrorInvalidValue;
  ((n == Ns + 1 ? (e = table_n<Ns + 1>(b, lds, tokens, canon, list, s), 0) : 0), ...);
  return e;
}

hipError_t launch_ngram_table(const NgramPartBatch& b, int max_slots, const int32_t* tokens, int n,
                              uint16_t* canon, uint2* list, hipStream_t s) {
  if (b.count <= 0) return hipSuccess;
  KernelTimer t(K_NGRAM_TABLE, s);
  return table_dispatch(std::make_integer_sequence<int, kMaxN>{}, n, b, ngram_table_lds(max_slots), tokens, canon,
                        list, s);
}

hipError_t launch_ngram_count(const NgramPartBatch& b, int total_blocks, int max_slots,
                              const int32_t* history, const int32_t* tokens, const uint2* list, int n,
                              uint16_t* partial, hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  const size_t lds = ngram_count_lds(max_slots, n);
  KernelTimer t(K_NGRAM_COUNT, s);
  return count_dispatch(std::make_integer_sequence<int, kMaxN>{}, n, b, total_blocks, lds, history, tokens, list,
                        partial, s);
}

hipError_t launch_ngram_weight(const NgramEpBatch& b, int total_blocks, int n, float w_min,
                               const uint16_t* partial, const uint16_t* canon, uint32_t* exposure,
                               float* weights, hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  KernelTimer t(K_NGRAM_WEIGHT, s);
  hipLaunchKernelGGL(ngram_weight_kernel, dim3(total_blocks), dim3(1024), 0, s, b, n, w_min, partial, canon,
                     exposure, weights);
  return hipGetLastError();
}

}  // namespace attt
