// Persistent n-gram counts of an episode's history (the history update of Algorithm 1:
// H^tok_{k+1} = H^tok_k followed by x_k) and exposure weights read from them (Eq. 8-9).
//
// A set is one caller-owned device buffer: a 256-byte header (history length, distinct n-grams
// held, error flags, the last n-1 history tokens (double-buffered), and the n and table size it
// was built for) followed by S slot records of R = 12 + 4n bytes rounded up to 16:
//   u64 key   64-bit key of the n-gram, 0 = empty slot (keys are odd)
//   u32 count occurrences of the n-gram in the history
//   i32 tok[n] the n-gram's tokens, for exact confirmation
// so a lookup reads one record (one or two cache lines) instead of three arrays. S is a power
// of two at least twice the capacity; slots are found by linear probing.
//
// Appending x to H adds the n-grams whose last token lies in x: those inside x and the n-1
// that start in the history's last n-1 tokens (n-grams straddling two updates count). One
// thread per new n-gram claims an empty slot with a 64-bit compare-and-swap on the key or
// finds its key, and adds 1 to the count; counts are integers, so the final table does not
// depend on the order of the adds. A second kernel confirms, after all claims have landed,
// that every new n-gram's slot holds exactly its tokens (two different n-grams with the same
// 64-bit key would otherwise share a count) and flags a collision if not; its last block to
// finish advances the history length and switches to the new tail.
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
  uint32_t ticket;  // blocks of the running confirm pass that have finished
};
static_assert(sizeof(NgramSetHeader) <= 256, "header fits its 256 bytes");

constexpr uint32_t kSetOverflow = 1u, kSetCollision = 2u, kSetMismatch = 4u;

__host__ __device__ __forceinline__ int64_t set_record_bytes(int n) { return (12 + 4 * n + 15) / 16 * 16; }

// Slot records: key at +0, count at +8, tokens from +12.
struct SetView {
  NgramSetHeader* hdr;
  uint8_t* rec;
  int64_t R;
  __device__ __forceinline__ unsigned long long* key(int64_t s) const {
    return reinterpret_cast<unsigned long long*>(rec + s * R);
  }
  __device__ __forceinline__ uint32_t* count(int64_t s) const { return reinterpret_cast<uint32_t*>(rec + s * R + 8); }
  __device__ __forceinline__ int32_t* toks(int64_t s) const { return reinterpret_cast<int32_t*>(rec + s * R + 12); }
};

__device__ __forceinline__ SetView set_view(uint8_t* base, int n) {
  SetView v;
  v.hdr = reinterpret_cast<NgramSetHeader*>(base);
  v.rec = base + 256;
  v.R = set_record_bytes(n);
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
  SetView v = set_view(static_cast<uint8_t*>(b.j[ji].set), n);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < S; i += (int64_t)gridDim.x * 256) {
    *v.key(i) = 0ull;
    *v.count(i) = 0u;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    v.hdr->ntok = 0;
    v.hdr->nent = 0;
    v.hdr->flags = 0;
    v.hdr->n = n;
    v.hdr->par = 0;
    v.hdr->slots = S;
    v.hdr->ticket = 0;
  }
}

// ---- append: count the new n-grams; the new tail goes to the other tail buffer ----------------
__global__ __launch_bounds__(256) void ngram_set_append_kernel(NgramSetBatch b, const int32_t* __restrict__ tokens,
                                                               int64_t S, int64_t capacity, int n) {
  int ji = 0;
  while (ji + 1 < b.count && b.j[ji + 1].block_begin <= (int)blockIdx.x) ++ji;
  const NgramSetJob J = b.j[ji];
  SetView v = set_view(static_cast<uint8_t*>(J.set), n);
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
    unsigned long long k = *v.key(slot);
    if (k == 0ull) {
      k = atomicCAS(v.key(slot), 0ull, key);
      if (k == 0ull) {  // claimed: store the tokens, count one occurrence and one entry
        int32_t* dst = v.toks(slot);
        for (int i = 0; i < n; ++i) dst[i] = t[i];
        atomicAdd(v.count(slot), 1u);
        if (atomicAdd(&v.hdr->nent, 1u) >= (uint64_t)capacity) atomicOr(&v.hdr->flags, kSetOverflow);
        return;
      }
    }
    if (k == key) {
      atomicAdd(v.count(slot), 1u);
      return;
    }
  }
  atomicOr(&v.hdr->flags, kSetOverflow);  // every slot taken
}

// ---- confirm: each new n-gram's slot holds its own tokens; the last block commits ----------------
// The block that finishes last (a ticket in the header, taken after a fence) advances the history
// length and switches to the new tail, once every block has read the old ones.
__global__ __launch_bounds__(256) void ngram_set_confirm_kernel(NgramSetBatch b, const int32_t* __restrict__ tokens,
                                                                int64_t S, int n) {
  int ji = 0;
  while (ji + 1 < b.count && b.j[ji + 1].block_begin <= (int)blockIdx.x) ++ji;
  const NgramSetJob J = b.j[ji];
  SetView v = set_view(static_cast<uint8_t*>(J.set), n);
  NgramSetHeader& h = *v.hdr;
  if (h.n != n || h.slots != S) return;  // uniform per block: the set is flagged, nothing commits
  const int e = ((int)blockIdx.x - J.block_begin) * 256 + threadIdx.x;
  int32_t t[kMaxN];
  if (e < J.L && gather_new(h, h.tail[h.par], tokens + J.tok_base, e, n, t)) {
    const unsigned long long key = set_key(t, n);
    int64_t slot = set_home(key, S);
    for (int64_t probe = 0; probe < S; ++probe, slot = (slot + 1) & (S - 1)) {
      const unsigned long long k = *v.key(slot);
      if (k == 0ull) break;  // not inserted: the table overflowed (already flagged)
      if (k == key) {
        bool same = true;
        const int32_t* st = v.toks(slot);
        for (int i = 0; i < n; ++i) same &= st[i] == t[i];
        if (!same) atomicOr(&h.flags, kSetCollision);
        break;
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    const uint32_t nb = (uint32_t)((J.L + 255) / 256);
    if (atomicAdd(&h.ticket, 1u) == nb - 1) {
      h.ntok += J.L;
      h.par ^= 1;
      h.ticket = 0;
    }
  }
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
  SetView v = set_view(static_cast<uint8_t*>(J.set), n);
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
        const unsigned long long k = *v.key(slot);
        if (k == 0ull) break;
        if (k == key) {
          bool same = true;
          const int32_t* st = v.toks(slot);
          for (int i = 0; i < n; ++i) same &= st[i] == t[i];
          if (same) cnt = *v.count(slot);
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
  const size_t raw = 256 + (size_t)S * (size_t)set_record_bytes(n);
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
    return hipGetLastError();
  }
  return hipSuccess;  // every text empty: nothing changes
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
