// n-gram exposure and token weights (Sec. 3.3, Eq. 8-9) on gfx950.
//
// Only the n-grams of the new update x_k matter for f, so the hash set is built over them
// (the small side: at most kQMax start positions per partition) and the history H^tok_k (the
// large side) is streamed once, coalesced, by many workgroups. Two kernels:
//
//   ngram_count_kernel   one workgroup per (partition, history chunk). It builds an LDS
//                        open-addressing table of the partition's query n-grams (32-bit
//                        entries: hash tag | first query position; a probe hit is confirmed
//                        by comparing all n tokens), hashes every history n-gram of its chunk
//                        from an LDS tile, counts hits with LDS atomics, and writes for every
//                        query position of the partition the count of its n-gram in the
//                        chunk (16 bits; a chunk has at most 65535 positions).
//   ngram_weight_kernel  per update token j: sums the chunk counts of the n-gram starts that
//                        cover j in a fixed order, f(j) = their maximum, and
//                        w = max(w_min, 1 / (1 + f)) with a correctly rounded division.
//
// No global atomics and no table in global memory: each workgroup's table lives only in its
// LDS, and its slot layout (which depends on insertion order) never leaves the workgroup.
// Results are integers, so f and w are bit-reproducible.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

constexpr uint32_t kEmpty = 0xFFFFFFFFu;  // tag field of a real entry never has bit 19 set
constexpr int kHistTile = 1984;  // two workgroups of 1024 threads fit in the 160 KiB LDS

__device__ __forceinline__ uint32_t ngram_hash(const int32_t* t, int n) {
  uint32_t h = 0x9E3779B9u ^ (uint32_t)n;
  for (int i = 0; i < n; ++i) {
    h ^= (uint32_t)t[i];
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
  }
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

__device__ __forceinline__ bool ngram_equal(const int32_t* a, const int32_t* b, int n) {
  for (int i = 0; i < n; ++i)
    if (a[i] != b[i]) return false;
  return true;
}

// Table entry: bits 31..12 hash tag (bit 31 always 0), bits 11..0 query position.
__device__ __forceinline__ uint32_t entry_of(uint32_t h, int q) { return ((h >> 1) & 0x7FFFF000u) | (uint32_t)q; }

__global__ __launch_bounds__(1024) void ngram_count_kernel(NgramPartBatch batch,
                                                           const int32_t* __restrict__ history,
                                                           const int32_t* __restrict__ tokens,
                                                           int n, uint16_t* __restrict__ partial) {
  int pi = 0;
  while (pi + 1 < batch.count && batch.p[pi + 1].chunk_begin <= (int)blockIdx.x) ++pi;
  const NgramPart P = batch.p[pi];
  const int c = (int)blockIdx.x - P.chunk_begin;
  const int64_t per = (P.hist_ngrams + P.chunks - 1) / P.chunks;
  const int64_t i0 = (int64_t)c * per;
  const int64_t i1 = min((int64_t)P.hist_ngrams, i0 + per);

  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* tab = reinterpret_cast<uint32_t*>(smem);   // [slots]
  uint32_t* cnt = tab + P.slots;                       // [slots / 2], two 16-bit counters per word
  uint16_t* qslot = reinterpret_cast<uint16_t*>(cnt + P.slots / 2);  // [kQMax]
  int32_t* xs = reinterpret_cast<int32_t*>(qslot + kQMax);           // [kQMax + 16]
  int32_t* ht = xs + kQMax + 16;                                     // [kHistTile + 16]

  const uint32_t mask = (uint32_t)P.slots - 1u;
  const int32_t* x = tokens + P.tok_base + P.q0;
  for (int i = threadIdx.x; i < P.slots; i += blockDim.x) tab[i] = kEmpty;
  for (int i = threadIdx.x; i < P.slots / 2; i += blockDim.x) cnt[i] = 0u;
  for (int i = threadIdx.x; i < P.qn + n - 1; i += blockDim.x) xs[i] = x[i];
  __syncthreads();
  // insert the partition's query n-grams; duplicates share the first inserted entry
  for (int q = threadIdx.x; q < P.qn; q += blockDim.x) {
    const uint32_t h = ngram_hash(xs + q, n);
    const uint32_t mine = entry_of(h, q);
    uint32_t slot = h & mask;
    while (true) {
      const uint32_t cur = atomicCAS(tab + slot, kEmpty, mine);
      if (cur == kEmpty) break;
      if ((cur & 0xFFFFF000u) == (mine & 0xFFFFF000u) && ngram_equal(xs + (cur & 0xFFFu), xs + q, n)) break;
      slot = (slot + 1u) & mask;
    }
    qslot[q] = (uint16_t)slot;
  }
  const int32_t* hist = history + P.hist_base;
  for (int64_t base = i0; base < i1; base += kHistTile) {
    const int m = (int)min((int64_t)kHistTile, i1 - base);
    __syncthreads();  // table complete (first pass) / previous tile consumed
    for (int i = threadIdx.x; i < m + n - 1; i += blockDim.x) ht[i] = hist[base + i];
    __syncthreads();
    for (int k = threadIdx.x; k < m; k += blockDim.x) {
      const int32_t* g = ht + k;
      const uint32_t h = ngram_hash(g, n);
      const uint32_t tag = entry_of(h, 0);
      uint32_t slot = h & mask;
      while (true) {
        const uint32_t e = tab[slot];
        if (e == kEmpty) break;
        if ((e & 0xFFFFF000u) == tag && ngram_equal(xs + (e & 0xFFFu), g, n)) {
          atomicAdd(cnt + (slot >> 1), 1u << ((slot & 1u) * 16u));
          break;
        }
        slot = (slot + 1u) & mask;
      }
    }
  }
  __syncthreads();
  uint16_t* out = partial + (P.chunk_begin_global + c) * (int64_t)kQMax;
  for (int q = threadIdx.x; q < P.qn; q += blockDim.x) {
    const uint32_t s = qslot[q];
    out[q] = (uint16_t)(cnt[s >> 1] >> ((s & 1u) * 16u));
  }
}

__global__ __launch_bounds__(256) void ngram_weight_kernel(NgramEpBatch batch, int n, float w_min,
                                                           const uint16_t* __restrict__ partial,
                                                           uint32_t* __restrict__ exposure,
                                                           float* __restrict__ weights) {
  int ei = 0;
  while (ei + 1 < batch.count && batch.e[ei + 1].block_begin <= (int)blockIdx.x) ++ei;
  const NgramEp E = batch.e[ei];
  const int j0 = ((int)blockIdx.x - E.block_begin) * 256;
  const int Q = E.L - n + 1;  // query start positions 0 .. Q-1
  __shared__ uint32_t cs[256 + kMaxN];
  // counts of the starts s in [j0 - n + 1, j0 + 255] that exist, summed over the history chunks
  const int s_lo = j0 - n + 1;
  for (int t = threadIdx.x; t < 256 + n - 1; t += blockDim.x) {
    const int s = s_lo + t;
    uint32_t total = 0;
    if (s >= 0 && s < Q) {
      const int p = s / kQMax;
      const uint16_t* col = partial + ((int64_t)E.chunk_base + (int64_t)p * E.chunks) * kQMax + (s - p * kQMax);
      for (int ch = 0; ch < E.chunks; ++ch) total += col[(int64_t)ch * kQMax];
    }
    cs[t] = total;
  }
  __syncthreads();
  const int j = j0 + threadIdx.x;
  if (j >= E.L) return;
  uint32_t f = 0;
  for (int i = 0; i < n; ++i) f = max(f, cs[threadIdx.x + i]);  // starts j-n+1 .. j; absent ones hold 0
  const float w = fmaxf(w_min, __fdiv_rn(1.0f, 1.0f + (float)f));
  if (exposure) exposure[E.tok_base + j] = f;
  weights[E.tok_base + j] = w;
}

// ---------------------------------------------------------------------------------------
size_t ngram_count_lds(int slots, int n) {
  (void)n;
  return (size_t)slots * 4 + (size_t)slots * 2 + (size_t)kQMax * 2 + (size_t)(kQMax + 16) * 4 +
         (size_t)(kHistTile + 16) * 4;
}

hipError_t launch_ngram_count(const NgramPartBatch& b, int total_blocks, int max_slots,
                              const int32_t* history, const int32_t* tokens, int n,
                              uint16_t* partial, hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  const size_t lds = ngram_count_lds(max_slots, n);
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)ngram_count_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  KernelTimer t(K_NGRAM_COUNT, s);
  hipLaunchKernelGGL(ngram_count_kernel, dim3(total_blocks), dim3(1024), lds, s, b, history, tokens,
                     n, partial);
  return hipGetLastError();
}

hipError_t launch_ngram_weight(const NgramEpBatch& b, int total_blocks, int n, float w_min,
                               const uint16_t* partial, uint32_t* exposure, float* weights,
                               hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  KernelTimer t(K_NGRAM_WEIGHT, s);
  hipLaunchKernelGGL(ngram_weight_kernel, dim3(total_blocks), dim3(256), 0, s, b, n, w_min, partial,
                     exposure, weights);
  return hipGetLastError();
}

}  // namespace attt
