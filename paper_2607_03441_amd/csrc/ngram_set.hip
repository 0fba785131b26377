// Persistent n-gram counts of an episode's history (the history update of Algorithm 1:
// H^tok_{k+1} = H^tok_k followed by x_k) and exposure weights read from them (Eq. 8-9).
//
// A set is one caller-owned device buffer:
//   header (256 B)  history length, distinct n-grams held, error flags, the last n-1 history
//                   tokens (double-buffered), and the n and table size it was built for
//   keys   u64 [S]  64-bit key of the n-gram in each slot, 0 = empty (keys are odd)
//   counts u32 [S]  occurrences of that n-gram in the history
//   toks   i32 [S][n] the n-gram's tokens, for exact confirmation
// S is a power of two at least twice the capacity; slots are found by linear probing.
//
// Appending x to H adds the n-grams whose last token lies in x: those inside x and the n-1
// that start in the history's last n-1 tokens (n-grams straddling two updates count). One
// thread per new n-gram claims an empty slot with a 64-bit compare-and-swap on the key or
// finds its key, and adds 1 to the count; counts are integers, so the final table does not
// depend on the order of the adds. A second kernel confirms, after all claims have landed,
// that every new n-gram's slot holds exactly its tokens (two different n-grams with the same
// 64-bit key would otherwise share a count) and flags a collision if not; a third advances
// the history length and switches to the new tail.
//
// The weights kernel looks up each n-gram start s of x (count 0 when absent or when the slot's
// tokens differ), then f(j) = max over the starts that cover j and w = max(w_min, 1/(1+f)),
// the same float32 division as the streaming path. A set whose flags are not clear (more
// distinct n-grams than its capacity, a key collision, or a call with another n or table size
// than the set was initialised for) yields f = 0xFFFFFFFF and w = NaN for every token.
#include <algorithm>

#include "common.hpp"
#include "internal.hpp"

namespace attt {

struct NgramSetHeader {
  int64_t ntok;     // history tokens appended so far
  uint32_t nent;    // distinct n-grams held
  uint32_t flags;   // kSetOverflow | kSetCollision | kSetMismatch
  int32_t n;        // n the set was initialised for
  int32_t par;      // which tail buffer is current
  int64_t slots;    // S
  int32_t tail[2][kMaxN];  // tail[par][i] = H[ntok - (n-1) + i] for the last min(ntok, n-1)
};
static_assert(sizeof(NgramSetHeader) <= 256, "header fits its 256 bytes");

constexpr uint32_t kSetOverflow = 1u, kSetCollision = 2u, kSetMismatch = 4u;

struct SetView {
  NgramSetHeader* hdr;
  unsigned long long* keys;
  uint32_t* counts;
  int32_t* toks;
};

__device__ __forceinline__ SetView set_view(uint8_t* base, int64_t S) {
  SetView v;
  v.hdr = reinterpret_cast<NgramSetHeader*>(base);
  v.keys = reinterpret_cast<unsigned long long*>(base + 256);
  v.counts = reinterpret_cast<uint32_t*>(base + 256 + S * 8);
  v.toks = reinterpret_cast<int32_t*>(base + 256 + S * 12);
  return v;
}

// 64-bit key of n tokens: a multiply-xorshift chain over the tokens and a final mix; forced
// odd so that 0 marks an empty slot. Equal keys are confirmed against the stored tokens.
__device__ __forceinline__ unsigned long long set_key(const int32_t* t, int n) {
  unsigned long long h = 0x243F6A8885A308D3ull ^ (unsigned long long)n;
  for (int i = 0; i < n; ++i) {
    h = (h ^ (unsigned long long)(uint32_t)t[i]) * 0x9E3779B97F4A7C15ull;
    h ^= h >> 29;
  }
  h ^= h >> 32;
  h *= 0xD6E8FEB86659FD93ull;
  h ^= h >> 32;
  return h | 1ull;
}

__device__ __forceinline__ int64_t set_home(unsigned long long key, int64_t S) {
  return (int64_t)((key >> 17) & (unsigned long long)(S - 1));
}

// The n tokens of the new n-gram whose last token is x[e]: positions ntok + e - n + 1 + i of
// the history followed by x; those before ntok come from the tail. False when the n-gram
// would start before the history's first token.
__device__ __forceinline__ bool gather_new(const NgramSetHeader& h, const int32_t* tail,
                                           const int32_t* x, int e, int n, int32_t* t) {
  const int64_t first = h.ntok + e - n + 1;
  if (first < 0) return false;
  for (int i = 0; i < n; ++i) {
    const int64_t p = first + i;
    t[i] = p < h.ntok ? tail[(int)(p - (h.ntok - (n - 1)))] : x[p - h.ntok];
  }
  return true;
}

// ---- init: empty table, empty history ---------------------------------------------------------
__global__ __launch_bounds__(256) void ngram_set_init_kernel(NgramSetBatch b, int64_t S, int n) {
  const int ji = (int)blockIdx.y;
  if (ji >= b.count) return;
  SetView v = set_view(static_cast<uint8_t*>(b.j[ji].set), S);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < S; i += (int64_t)gridDim.x * 256) {
    v.keys[i] = 0ull;
    v.counts[i] = 0u;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    v.hdr->ntok = 0;
    v.hdr->nent = 0;
    v.hdr->flags = 0;
    v.hdr->n = n;
    v.hdr->par = 0;
    v.hdr->slots = S;
  }
}

// ---- append: count the new n-grams; the new tail goes to the other tail buffer ----------------
__global__ __launch_bounds__(256) void ngram_set_append_kernel(NgramSetBatch b, const int32_t* __restrict__ tokens,
                                                               int64_t S, int64_t capacity, int n) {
  int ji = 0;
  while (ji + 1 < b.count && b.j[ji + 1].block_begin <= (int)blockIdx.x) ++ji;
  const NgramSetJob J = b.j[ji];
  SetView v = set_view(static_cast<uint8_t*>(J.set), S);
  const NgramSetHeader& h = *v.hdr;
  if (h.n != n || h.slots != S) {
    if (blockIdx.x == J.block_begin && threadIdx.x == 0) atomicOr(&v.hdr->flags, kSetMismatch);
    return;
  }
  const int e = ((int)blockIdx.x - J.block_begin) * 256 + threadIdx.x;
  if (e >= J.L) return;
  const int32_t* x = tokens + J.tok_base;
  const int32_t* tail = h.tail[h.par];
  // new tail: the last n-1 tokens of (history, x), oldest first
  const int keep = n - 1;
  if (e >= J.L - keep) {
    const int i = keep - (J.L - e);  // this token's place in the new tail
    v.hdr->tail[h.par ^ 1][i] = x[e];
  }
  if (J.L < keep && e == 0) {  // x shorter than the tail: the older tail entries shift down
    for (int i = 0; i < keep - J.L; ++i) v.hdr->tail[h.par ^ 1][i] = tail[i + J.L];
  }
  int32_t t[kMaxN];
  if (!gather_new(h, tail, x, e, n, t)) return;
  const unsigned long long key = set_key(t, n);
  int64_t slot = set_home(key, S);
  for (int64_t probe = 0; probe < S; ++probe, slot = (slot + 1) & (S - 1)) {
    unsigned long long k = v.keys[slot];
    if (k == 0ull) {
      k = atomicCAS(v.keys + slot, 0ull, key);
      if (k == 0ull) {  // claimed: store the tokens, count one occurrence and one entry
        for (int i = 0; i < n; ++i) v.toks[slot * n + i] = t[i];
        atomicAdd(v.counts + slot, 1u);
        if (atomicAdd(&v.hdr->nent, 1u) >= (uint64_t)capacity) atomicOr(&v.hdr->flags, kSetOverflow);
        return;
      }
    }
    if (k == key) {
      atomicAdd(v.counts + slot, 1u);
      return;
    }
  }
  atomicOr(&v.hdr->flags, kSetOverflow);  // every slot taken
}

// ---- confirm: each new n-gram's slot holds its own tokens ---------------------------------------
__global__ __launch_bounds__(256) void ngram_set_confirm_kernel(NgramSetBatch b, const int32_t* __restrict__ tokens,
                                                                int64_t S, int n) {
  int ji = 0;
  while (ji + 1 < b.count && b.j[ji + 1].block_begin <= (int)blockIdx.x) ++ji;
  const NgramSetJob J = b.j[ji];
  SetView v = set_view(static_cast<uint8_t*>(J.set), S);
  const NgramSetHeader& h = *v.hdr;
  if (h.n != n || h.slots != S) return;
  const int e = ((int)blockIdx.x - J.block_begin) * 256 + threadIdx.x;
  if (e >= J.L) return;
  int32_t t[kMaxN];
  if (!gather_new(h, h.tail[h.par], tokens + J.tok_base, e, n, t)) return;
  const unsigned long long key = set_key(t, n);
  int64_t slot = set_home(key, S);
  for (int64_t probe = 0; probe < S; ++probe, slot = (slot + 1) & (S - 1)) {
    const unsigned long long k = v.keys[slot];
    if (k == 0ull) return;  // not inserted: the table overflowed (already flagged)
    if (k == key) {
      bool same = true;
      for (int i = 0; i < n; ++i) same &= v.toks[slot * n + i] == t[i];
      if (!same) atomicOr(&v.hdr->flags, kSetCollision);
      return;
    }
  }
}

// ---- commit: history length and tail move on (one thread per set) --------------------------------
__global__ __launch_bounds__(64) void ngram_set_commit_kernel(NgramSetBatch b, int64_t S, int n) {
  const int ji = (int)(blockIdx.x * 64 + threadIdx.x);
  if (ji >= b.count) return;
  SetView v = set_view(static_cast<uint8_t*>(b.j[ji].set), S);
  if (v.hdr->n != n || v.hdr->slots != S || b.j[ji].L == 0) return;  // an empty x keeps the tail
  v.hdr->ntok += b.j[ji].L;
  v.hdr->par ^= 1;
}

// ---- weights: lookups of x's n-gram starts, window maximum, w -------------------------------------
// A block covers 256 positions j0 .. j0+255 of one update; it looks up the starts
// j0-n+1 .. j0+255 into LDS (recomputing the n-1 starts it shares with the previous block).
__global__ __launch_bounds__(256) void ngram_set_weights_kernel(NgramSetBatch b, const int32_t* __restrict__ tokens,
                                                                int64_t S, int n, float w_min,
                                                                uint32_t* __restrict__ exposure,
                                                                float* __restrict__ weights) {
  int ji = 0;
  while (ji + 1 < b.count && b.j[ji + 1].block_begin <= (int)blockIdx.x) ++ji;
  const NgramSetJob J = b.j[ji];
  SetView v = set_view(static_cast<uint8_t*>(J.set), S);
  const bool bad = v.hdr->flags != 0 || v.hdr->n != n || v.hdr->slots != S;
  const int j0 = ((int)blockIdx.x - J.block_begin) * 256;
  const int32_t* x = tokens + J.tok_base;
  const int L = J.L;
  __shared__ uint32_t c[256 + kMaxN];
  for (int u = threadIdx.x; u < 256 + n - 1; u += 256) {
    const int s = j0 - (n - 1) + u;  // n-gram start
    uint32_t cnt = 0;
    if (!bad && s >= 0 && s + n <= L) {
      int32_t t[kMaxN];
      for (int i = 0; i < n; ++i) t[i] = x[s + i];
      const unsigned long long key = set_key(t, n);
      int64_t slot = set_home(key, S);
      for (int64_t probe = 0; probe < S; ++probe, slot = (slot + 1) & (S - 1)) {
        const unsigned long long k = v.keys[slot];
        if (k == 0ull) break;
        if (k == key) {
          bool same = true;
          for (int i = 0; i < n; ++i) same &= v.toks[slot * n + i] == t[i];
          if (same) cnt = v.counts[slot];
          break;
        }
      }
    }
    c[u] = cnt;
  }
  __syncthreads();
  const int j = j0 + threadIdx.x;
  if (j >= L) return;
  uint32_t f = 0;
  for (int i = 0; i < n; ++i) f = max(f, c[threadIdx.x + i]);  // starts j-n+1 .. j
  float w = fmaxf(w_min, __fdiv_rn(1.0f, 1.0f + (float)f));
  if (bad) {
    f = 0xFFFFFFFFu;
    w = __int_as_float(0x7FC00000);
  }
  if (exposure) exposure[J.tok_base + j] = f;
  weights[J.tok_base + j] = w;
}

size_t ngram_set_bytes(int64_t S, int n) {
  const size_t raw = 256 + (size_t)S * (8 + 4) + (size_t)S * n * 4;
  return (raw + 255) & ~(size_t)255;
}

hipError_t launch_ngram_set_init(const NgramSetBatch& b, int64_t S, int n, hipStream_t s) {
  KernelTimer t(K_NGRAM_SET, s);
  const int gx = (int)std::min<int64_t>(1024, (S + 255) / 256);
  hipLaunchKernelGGL(ngram_set_init_kernel, dim3(gx, b.count), dim3(256), 0, s, b, S, n);
  return hipGetLastError();
}

hipError_t launch_ngram_set_append(const NgramSetBatch& b, int blocks, const int32_t* tokens, int64_t S,
                                   int64_t capacity, int n, hipStream_t s) {
  KernelTimer t(K_NGRAM_SET, s);
  if (blocks > 0) {
    hipLaunchKernelGGL(ngram_set_append_kernel, dim3(blocks), dim3(256), 0, s, b, tokens, S, capacity, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(ngram_set_confirm_kernel, dim3(blocks), dim3(256), 0, s, b, tokens, S, n);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ngram_set_commit_kernel, dim3((b.count + 63) / 64), dim3(64), 0, s, b, S, n);
  return hipGetLastError();
}

hipError_t launch_ngram_set_weights(const NgramSetBatch& b, int blocks, const int32_t* tokens, int64_t S,
                                    int n, float w_min, uint32_t* exposure, float* weights, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_NGRAM_SET_WEIGHT, s);
  hipLaunchKernelGGL(ngram_set_weights_kernel, dim3(blocks), dim3(256), 0, s, b, tokens, S, n, w_min,
                     exposure, weights);
  return hipGetLastError();
}

}  // namespace attt
