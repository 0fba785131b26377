// n-gram exposure and token weights (Sec. 3.3, Eq. 8-9) on gfx950.
//
// Only the n-grams of the new update x_k matter for f, so the hash set is built over them
// (the small side: at most kQMax start positions per partition) and the history H^tok_k (the
// large side) is streamed once, coalesced, by many workgroups. Two kernels:
//
//   ngram_count_kernel   one workgroup per (partition, history chunk). It builds an LDS table
//                        of the partition's query n-grams in buckets of four 32-bit entries
//                        (hash tag | first query position with that n-gram), hashes every
//                        history n-gram of its chunk from a double-buffered LDS tile, looks it
//                        up with one 16-byte LDS read per bucket (a tag match is confirmed by
//                        comparing all n tokens), counts hits per first query position with
//                        LDS atomics, and writes for every query position of the partition the
//                        count of its n-gram in the chunk (16 bits; a chunk has at most 65535
//                        positions).
//   ngram_weight_kernel  per update token j: sums the chunk counts of the n-gram starts that
//                        cover j in a fixed order, f(j) = their maximum, and
//                        w = max(w_min, 1 / (1 + f)) with a correctly rounded division.
//
// No global atomics and no table in global memory: each workgroup's table lives only in its
// LDS, and which query position stands for a repeated n-gram (insertion order) never leaves
// the workgroup. Results are integers, so f and w are bit-reproducible.
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
constexpr int kHistTile = 1984;           // positions per history tile (two tiles per workgroup)
constexpr int kHalo = 16;                 // >= n - 1 extra tokens after a tile

// Hash of n tokens held in registers (n is a compile-time constant of the kernel). Full-rate
// 24-bit multiply-adds (v_mad_u32_u24) fold each token in; the high bits re-enter through the
// shifted term. Only table placement depends on it: every tag match is verified token by token.
template <int N>
__device__ __forceinline__ uint32_t ngram_hash(const int32_t (&t)[N]) {
  uint32_t h = 0x9E3779B9u ^ (uint32_t)N;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    h ^= (uint32_t)t[i];
    h = __umul24(h, 0x2F6B9Du) + (h >> 9);
  }
  h ^= h >> 15;
  h = __umul24(h, 0x3C6EF3u) + (h >> 11);
  h ^= h >> 16;
  return h;
}

template <int N>
__device__ __forceinline__ void ngram_load(const int32_t* p, int32_t (&t)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) t[i] = p[i];
}

// All n comparisons from independent loads.
template <int N>
__device__ __forceinline__ bool ngram_equal(const int32_t* a, const int32_t (&t)[N]) {
  bool eq = true;
#pragma unroll
  for (int i = 0; i < N; ++i) eq &= a[i] == t[i];
  return eq;
}

// Table entry: bits 31..12 hash tag (bit 31 always 0), bits 11..0 query position. The bucket
// index takes the hash's low bits, the tag its high bits.
__device__ __forceinline__ uint32_t entry_of(uint32_t h, int q) { return ((h >> 1) & 0x7FFFF000u) | (uint32_t)q; }
constexpr uint32_t kTagMask = 0xFFFFF000u;
constexpr int kDepth = 4;  // history tiles in flight per workgroup (register stages)

template <int N>
__global__ __launch_bounds__(1024) void ngram_count_kernel(NgramPartBatch batch,
                                                           const int32_t* __restrict__ history,
                                                           const int32_t* __restrict__ tokens,
                                                           uint16_t* __restrict__ partial) {
  int pi = 0;
  while (pi + 1 < batch.count && batch.p[pi + 1].chunk_begin <= (int)blockIdx.x) ++pi;
  const NgramPart P = batch.p[pi];
  const int c = (int)blockIdx.x - P.chunk_begin;
  const int64_t per = (P.hist_ngrams + P.chunks - 1) / P.chunks;
  const int64_t i0 = (int64_t)c * per;
  const int64_t i1 = min((int64_t)P.hist_ngrams, i0 + per);
  const int ntiles = i1 > i0 ? (int)((i1 - i0 + kHistTile - 1) / kHistTile) : 0;

  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* tab = reinterpret_cast<uint32_t*>(smem);                 // [slots], 4 per bucket
  uint32_t* cnt = tab + P.slots;                                     // [kQMax / 2], 16-bit pairs
  uint16_t* canon = reinterpret_cast<uint16_t*>(cnt + kQMax / 2);    // [kQMax]
  int32_t* xs = reinterpret_cast<int32_t*>(canon + kQMax);           // [kQMax + kHalo]
  int32_t* ht = xs + kQMax + kHalo;                                  // [2][kHistTile + kHalo]

  const uint32_t bmask = (uint32_t)(P.slots >> 2) - 1u;
  const int32_t* x = tokens + P.tok_base + P.q0;
  const int32_t* hist = history + P.hist_base;
  const int tid = threadIdx.x;
  // History tiles travel through kDepth register stages: tile k is loaded while tile k-kDepth
  // is hashed, then stored to the LDS buffer k&1 one iteration before it is hashed.
  // The chunk's history with its n-1 token halo is [i0, i1 + N - 1): the descriptor covers
  // exactly that range, so loads past its end return zero without a branch.
  constexpr int kPer = (kHistTile + kHalo + 1023) / 1024;  // loads per thread per tile
  const __amdgpu_buffer_rsrc_t rh =
      buffer_rsrc(hist + i0, i1 > i0 ? (int)((i1 - i0 + N - 1) * 4) : 0);
  // the partition's query tokens (qn + N - 1 of them) go to registers first, so that waiting
  // for them later does not wait for the history tiles issued after them
  constexpr int kXPer = (kQMax + kHalo + 1023) / 1024;
  const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(x, (P.qn + N - 1) * 4);
  int32_t xv[kXPer];
#pragma unroll
  for (int u = 0; u < kXPer; ++u)
    xv[u] = __builtin_amdgcn_raw_buffer_load_b32(rx, (uint32_t)(tid + u * 1024) * 4u, 0, 0);
  int32_t pre[kDepth][kPer];
  auto fetch = [&](int k, int32_t (&r)[kPer]) {
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      r[u] = __builtin_amdgcn_raw_buffer_load_b32(rh, (uint32_t)(k * kHistTile + tid + u * 1024) * 4u, 0, 0);
  };
  auto stash = [&](int buf, const int32_t (&r)[kPer]) {
    int32_t* dst = ht + buf * (kHistTile + kHalo);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int i = tid + u * 1024;
      if (i < kHistTile + kHalo) dst[i] = r[u];
    }
  };
#pragma unroll
  for (int k = 0; k < kDepth; ++k) fetch(k, pre[k]);

  for (int i = tid; i < P.slots; i += 1024) tab[i] = kEmpty;
  for (int i = tid; i < kQMax / 2; i += 1024) cnt[i] = 0u;
#pragma unroll
  for (int u = 0; u < kXPer; ++u)
    if (tid + u * 1024 < kQMax + kHalo) xs[tid + u * 1024] = xv[u];
  __syncthreads();
  // Insert the partition's query n-grams. Slots of a bucket are claimed in order, so the
  // occupied slots of every bucket always form a prefix and a bucket with a free slot ends
  // every search. A repeated n-gram resolves to the entry inserted first.
  for (int q = tid; q < P.qn; q += 1024) {
    int32_t t[N];
    ngram_load(xs + q, t);
    const uint32_t h = ngram_hash(t);
    const uint32_t mine = entry_of(h, q);
    uint32_t b = h & bmask;
    int who = -1;
    while (who < 0) {
#pragma unroll
      for (int sidx = 0; sidx < 4 && who < 0; ++sidx) {
        const uint32_t cur = atomicCAS(tab + b * 4 + sidx, kEmpty, mine);
        if (cur == kEmpty) who = q;
        else if ((cur & kTagMask) == (mine & kTagMask) && ngram_equal(xs + (cur & 0xFFFu), t))
          who = (int)(cur & 0xFFFu);
      }
      b = (b + 1u) & bmask;
    }
    canon[q] = (uint16_t)who;
  }
  stash(0, pre[0]);
  __syncthreads();

  const u32x4* tab4 = reinterpret_cast<const u32x4*>(tab);
  auto hash_tile = [&](int k) {
    const int64_t base = i0 + (int64_t)k * kHistTile;
    const int m = (int)min((int64_t)kHistTile, i1 - base);
    const int32_t* cur = ht + (k & 1) * (kHistTile + kHalo);
    for (int j = tid; j < m; j += 1024) {
      int32_t t[N];
      ngram_load(cur + j, t);
      const uint32_t h = ngram_hash(t);
      const uint32_t tag = entry_of(h, 0);
      uint32_t b = h & bmask;
      while (true) {
        const u32x4 e = tab4[b];
        // slots whose tag matches; the first is verified, the others only if it fails
        uint32_t cand = 0;
#pragma unroll
        for (int sidx = 0; sidx < 4; ++sidx) cand |= (uint32_t)((e[sidx] & kTagMask) == tag) << sidx;
        int hit = -1;
        while (cand) {
          const int sidx = __builtin_ctz(cand);
          const uint32_t ent = sidx == 0 ? e[0] : sidx == 1 ? e[1] : sidx == 2 ? e[2] : e[3];
          if (ngram_equal(xs + (ent & 0xFFFu), t)) {
            hit = (int)(ent & 0xFFFu);
            break;
          }
          cand &= cand - 1u;
        }
        if (hit >= 0) {
          atomicAdd(cnt + (hit >> 1), 1u << ((hit & 1) * 16));
          break;
        }
        if (e[3] == kEmpty) break;  // bucket not full: the n-gram is not in the table
        b = (b + 1u) & bmask;
      }
    }
  };
  // Iteration k: load tile k + kDepth into the stage tile k left, hash tile k from LDS, store
  // tile k + 1 (loaded kDepth - 1 iterations ago) into the other LDS buffer, one barrier. The
  // stage indices are compile-time: the loop advances kDepth tiles per trip. Every trip issues
  // the same loads on every path (tiles past the chunk read as zero and hash no position), so
  // each store waits only for its own stage.
  for (int k0 = 0; k0 < ntiles; k0 += kDepth) {
#pragma unroll
    for (int u = 0; u < kDepth; ++u) {
      const int k = k0 + u;
      fetch(k + kDepth, pre[u]);
      hash_tile(k);
      stash((k + 1) & 1, pre[(u + 1) % kDepth]);
      __syncthreads();
    }
  }
  uint16_t* out = partial + (P.chunk_begin_global + c) * (int64_t)kQMax;
  for (int q = tid; q < P.qn; q += 1024) {
    const int r = canon[q];
    out[q] = (uint16_t)(cnt[r >> 1] >> ((r & 1) * 16));
  }
}

// 256 update tokens per block; the chunk counts of each n-gram start are summed by four
// groups of 256 threads (a quarter of the chunks each, several loads in flight per thread),
// then combined in LDS. Integer sums, so the order does not matter.
__global__ __launch_bounds__(1024) void ngram_weight_kernel(NgramEpBatch batch, int n, float w_min,
                                                            const uint16_t* __restrict__ partial,
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
    if (s >= 0 && s < Q) {
      const int p = s / kQMax;
      const uint16_t* col = partial + ((int64_t)E.chunk_base + (int64_t)p * E.chunks) * kQMax + (s - p * kQMax);
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
  return (size_t)slots * 4 + (size_t)kQMax * 2 + (size_t)kQMax * 2 + (size_t)(kQMax + kHalo) * 4 +
         (size_t)2 * (kHistTile + kHalo) * 4;
}

template <int N>
static hipError_t count_n(const NgramPartBatch& b, int total_blocks, size_t lds, const int32_t* history,
                          const int32_t* tokens, uint16_t* partial, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)ngram_count_kernel<N>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr = true;
  }
  hipLaunchKernelGGL(ngram_count_kernel<N>, dim3(total_blocks), dim3(1024), lds, s, b, history, tokens,
                     partial);
  return hipGetLastError();
}

template <int... Ns>
static hipError_t count_dispatch(std::integer_sequence<int, Ns...>, int n, const NgramPartBatch& b,
                                 int total_blocks, size_t lds, const int32_t* history,
                                 const int32_t* tokens, uint16_t* partial, hipStream_t s) {
  hipError_t e = hipErrorInvalidValue;
  ((n == Ns + 1 ? (e = count_n<Ns + 1>(b, total_blocks, lds, history, tokens, partial, s), 0) : 0), ...);
  return e;
}

hipError_t launch_ngram_count(const NgramPartBatch& b, int total_blocks, int max_slots,
                              const int32_t* history, const int32_t* tokens, int n,
                              uint16_t* partial, hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  const size_t lds = ngram_count_lds(max_slots, n);
  KernelTimer t(K_NGRAM_COUNT, s);
  return count_dispatch(std::make_integer_sequence<int, kMaxN>{}, n, b, total_blocks, lds, history, tokens,
                        partial, s);
}

hipError_t launch_ngram_weight(const NgramEpBatch& b, int total_blocks, int n, float w_min,
                               const uint16_t* partial, uint32_t* exposure, float* weights,
                               hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  KernelTimer t(K_NGRAM_WEIGHT, s);
  hipLaunchKernelGGL(ngram_weight_kernel, dim3(total_blocks), dim3(1024), 0, s, b, n, w_min, partial,
                     exposure, weights);
  return hipGetLastError();
}

}  // namespace attt
