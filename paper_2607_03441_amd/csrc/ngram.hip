// n-gram exposure and token weights (Sec. 3.3, Eq. 8-9) on gfx950.
//
// Only the n-grams of the new update x_k matter for f, so the hash set is built over
// them (the small side: at most kQMax start positions per partition, kept in LDS) and the
// history H^tok_k (the large side) is streamed past it once, coalesced, by many
// workgroups. Three kernels:
//   ngram_build_kernel   one workgroup per partition: insert the partition's query
//                        n-grams into an LDS open-addressing table with exact token
//                        verification, write the table out, zero the partition's
//                        counters and record, per query start s, the counter cell of its
//                        n-gram (duplicates inside x_k share one cell).
//   ngram_count_kernel   workgroups over (partition, history chunk): copy the table to
//                        LDS, hash every history n-gram of the chunk from an LDS tile,
//                        probe, verify tokens exactly and count hits with LDS atomics;
//                        flush non-zero counters with one global integer atomic each.
//   ngram_weight_kernel  per update token j: f(j) = max count over the n-grams that
//                        cover j (a window of n start positions), w = max(w_min, 1/(1+f)).
// Integer atomics only, so f and w are bit-reproducible. Keys are never reduced to a
// fingerprint: a probe hit is confirmed by comparing all n tokens.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

constexpr uint32_t kEmptyPos = 0xFFFFFFFFu;
constexpr unsigned long long kEmptySlot = 0xFFFFFFFF00000000ull;  // .x hash 0, .y pos empty
constexpr int kHistTile = 4096;

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

__global__ __launch_bounds__(1024) void ngram_build_kernel(NgramPartBatch batch,
                                                           const int32_t* __restrict__ tokens,
                                                           int n, uint2* __restrict__ tables,
                                                           uint32_t* __restrict__ counts,
                                                           uint32_t* __restrict__ qcell) {
  const NgramPart P = batch.p[blockIdx.x];
  extern __shared__ __align__(16) uint8_t smem[];
  uint2* tab = reinterpret_cast<uint2*>(smem);
  int32_t* xs = reinterpret_cast<int32_t*>(tab + P.slots);
  const int nt = P.qn + n - 1;
  const int32_t* x = tokens + P.tok_base + P.q0;
  for (int i = threadIdx.x; i < P.slots; i += blockDim.x) tab[i] = make_uint2(0u, kEmptyPos);
  for (int i = threadIdx.x; i < nt; i += blockDim.x) xs[i] = x[i];
  __syncthreads();
  const uint32_t mask = (uint32_t)P.slots - 1u;
  for (int s = threadIdx.x; s < P.qn; s += blockDim.x) {
    const uint32_t h = ngram_hash(xs + s, n);
    uint32_t slot = h & mask;
    const unsigned long long mine = ((unsigned long long)(uint32_t)s << 32) | h;
    while (true) {
      unsigned long long cur =
          atomicCAS(reinterpret_cast<unsigned long long*>(tab + slot), kEmptySlot, mine);
      if (cur == kEmptySlot) break;
      const uint32_t ch = (uint32_t)cur, cs = (uint32_t)(cur >> 32);
      if (ch == h && ngram_equal(xs + cs, xs + s, n)) break;
      slot = (slot + 1u) & mask;
    }
    qcell[P.tok_base + P.q0 + s] = P.count_off + slot;
  }
  __syncthreads();
  uint2* gt = tables + P.table_off;
  uint32_t* gc = counts + P.count_off;
  for (int i = threadIdx.x; i < P.slots; i += blockDim.x) {
    gt[i] = tab[i];
    gc[i] = 0u;
  }
}

__global__ __launch_bounds__(1024) void ngram_count_kernel(NgramPartBatch batch,
                                                           const int32_t* __restrict__ history,
                                                           const int32_t* __restrict__ tokens,
                                                           int n, const uint2* __restrict__ tables,
                                                           uint32_t* __restrict__ counts) {
  int pi = 0;
  while (pi + 1 < batch.count && batch.p[pi + 1].chunk_begin <= (int)blockIdx.x) ++pi;
  const NgramPart P = batch.p[pi];
  const int c = (int)blockIdx.x - P.chunk_begin;
  const int64_t per = (P.hist_ngrams + P.chunks - 1) / P.chunks;
  const int64_t i0 = (int64_t)c * per;
  const int64_t i1 = min((int64_t)P.hist_ngrams, i0 + per);
  if (i0 >= i1) return;  // uniform across the workgroup

  extern __shared__ __align__(16) uint8_t smem[];
  uint2* tab = reinterpret_cast<uint2*>(smem);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(tab + P.slots);
  int32_t* xs = reinterpret_cast<int32_t*>(cnt + P.slots);
  int32_t* ht = xs + ((P.qn + n - 1 + 3) & ~3);

  const uint2* gt = tables + P.table_off;
  for (int i = threadIdx.x; i < P.slots; i += blockDim.x) {
    tab[i] = gt[i];
    cnt[i] = 0u;
  }
  const int32_t* x = tokens + P.tok_base + P.q0;
  for (int i = threadIdx.x; i < P.qn + n - 1; i += blockDim.x) xs[i] = x[i];
  const int32_t* hist = history + P.hist_base;
  const uint32_t mask = (uint32_t)P.slots - 1u;

  for (int64_t base = i0; base < i1; base += kHistTile) {
    const int m = (int)min((int64_t)kHistTile, i1 - base);
    __syncthreads();  // previous tile fully consumed (and table ready on the first pass)
    for (int i = threadIdx.x; i < m + n - 1; i += blockDim.x) ht[i] = hist[base + i];
    __syncthreads();
    for (int k = threadIdx.x; k < m; k += blockDim.x) {
      const int32_t* g = ht + k;
      const uint32_t h = ngram_hash(g, n);
      uint32_t slot = h & mask;
      while (true) {
        const uint2 e = tab[slot];
        if (e.y == kEmptyPos) break;
        if (e.x == h && ngram_equal(xs + e.y, g, n)) {
          atomicAdd(cnt + slot, 1u);
          break;
        }
        slot = (slot + 1u) & mask;
      }
    }
  }
  __syncthreads();
  uint32_t* gc = counts + P.count_off;
  for (int i = threadIdx.x; i < P.slots; i += blockDim.x) {
    const uint32_t v = cnt[i];
    if (v) atomicAdd(gc + i, v);
  }
}

__global__ __launch_bounds__(256) void ngram_weight_kernel(NgramEpBatch batch, int n, float w_min,
                                                           const uint32_t* __restrict__ counts,
                                                           const uint32_t* __restrict__ qcell,
                                                           uint32_t* __restrict__ exposure,
                                                           float* __restrict__ weights) {
  int ei = 0;
  while (ei + 1 < batch.count && batch.e[ei + 1].block_begin <= (int)blockIdx.x) ++ei;
  const NgramEp E = batch.e[ei];
  const int j = ((int)blockIdx.x - E.block_begin) * blockDim.x + threadIdx.x;
  if (j >= E.L) return;
  const int Q = E.L - n + 1;  // query start positions 0 .. Q-1
  const int lo = max(0, j - n + 1);
  const int hi = min(j, Q - 1);
  uint32_t f = 0;
  for (int s = lo; s <= hi; ++s) f = max(f, counts[qcell[E.tok_base + s]]);
  const float w = fmaxf(w_min, __fdiv_rn(1.0f, 1.0f + (float)f));
  if (exposure) exposure[E.tok_base + j] = f;
  weights[E.tok_base + j] = w;
}

// ---------------------------------------------------------------------------------------
size_t ngram_build_lds(int slots, int n) { return (size_t)slots * 8 + (size_t)(kQMax + n) * 4; }

size_t ngram_count_lds(int slots, int n) {
  return (size_t)slots * 12 + (size_t)(((kQMax + n - 1 + 3) & ~3) + kHistTile + n) * 4;
}

hipError_t launch_ngram_build(const NgramPartBatch& b, int max_slots, const int32_t* tokens, int n,
                              uint2* tables, uint32_t* counts, uint32_t* qcell, hipStream_t s) {
  const size_t lds = ngram_build_lds(max_slots, n);
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)ngram_build_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  KernelTimer t(K_NGRAM_BUILD, s);
  hipLaunchKernelGGL(ngram_build_kernel, dim3(b.count), dim3(1024), lds, s, b, tokens, n, tables,
                     counts, qcell);
  return hipGetLastError();
}

hipError_t launch_ngram_count(const NgramPartBatch& b, int total_blocks, int max_slots,
                              const int32_t* history, const int32_t* tokens, int n,
                              const uint2* tables, uint32_t* counts, hipStream_t s) {
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
                     n, tables, counts);
  return hipGetLastError();
}

hipError_t launch_ngram_weight(const NgramEpBatch& b, int total_blocks, int n, float w_min,
                               const uint32_t* counts, const uint32_t* qcell, uint32_t* exposure,
                               float* weights, hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  KernelTimer t(K_NGRAM_WEIGHT, s);
  hipLaunchKernelGGL(ngram_weight_kernel, dim3(total_blocks), dim3(256), 0, s, b, n, w_min, counts,
                     qcell, exposure, weights);
  return hipGetLastError();
}

}  // namespace attt
