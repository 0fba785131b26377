// Update-text repetition (Sec. 3.2, Eq. 6-7): rho(x_k) = max over the previous update texts x'
// of the episode of the Jaccard similarity of the word sets W(x_k) and W(x'), nu = 1 - rho, and
// the sequence-level filter that skips an update when nu < tau.
//
//   rep_count_kernel   one 1024-thread workgroup per (previous text, hash partition). Words are
//                      split into `parts` partitions by the high bits of a 32-bit hash (the
//                      MurmurHash3 finalizer), so |A|, |B| and |A & B| are sums over partitions
//                      and a partition's sets fit LDS whatever the text lengths. The workgroup
//                      inserts its partition's words of the candidate into one LDS hash set and
//                      those of the previous text into another; a new entry of the second set
//                      that is also in the first counts towards the intersection.
//   rep_reduce_kernel  one thread per episode: sums the partitions, takes the maximum Jaccard
//                      over the previous texts by exact cross-multiplication (the first maximum
//                      wins a tie), rho = the nearest float64 to |A & B| / |A | B|,
//                      nu = RN(1 - rho), skip = nu < tau.
// Integer counts throughout, so the result is bit-reproducible.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

constexpr uint32_t kRepEmpty = 0xFFFFFFFFu;

__device__ __forceinline__ uint32_t word_hash(int32_t w) {
  uint32_t h = (uint32_t)w;
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}
// partition of a hash: multiply-shift range reduction of its high 24 bits
__device__ __forceinline__ int part_of(uint32_t h, int parts) { return (int)(((h >> 8) * (uint32_t)parts) >> 24); }

// Inserts w into the open-addressing set `tab` (kRepSlots entries, linear probing from the
// hash's low bits). Returns 1 if w was new, 0 if present, -1 if the set is full (every probe
// taken: the caller flags the call). The value kRepEmpty marks a free slot.
__device__ __forceinline__ int set_insert(uint32_t* tab, uint32_t h, uint32_t w) {
  uint32_t s = h & (kRepSlots - 1);
  for (int probe = 0; probe < kRepSlots; ++probe) {
    const uint32_t cur = atomicCAS(tab + s, kRepEmpty, w);
    if (cur == kRepEmpty) return 1;
    if (cur == w) return 0;
    s = (s + 1u) & (kRepSlots - 1);
  }
  return -1;
}
__device__ __forceinline__ bool set_contains(const uint32_t* tab, uint32_t h, uint32_t w) {
  uint32_t s = h & (kRepSlots - 1);
  for (int probe = 0; probe < kRepSlots; ++probe) {
    const uint32_t cur = tab[s];
    if (cur == w) return true;
    if (cur == kRepEmpty) return false;
    s = (s + 1u) & (kRepSlots - 1);
  }
  return false;
}

__global__ __launch_bounds__(1024) void rep_count_kernel(RepBatch batch, const int32_t* __restrict__ words,
                                                         const int64_t* __restrict__ toff,
                                                         int32_t* __restrict__ counts) {
  int ei = 0;
  while (ei + 1 < batch.count && batch.e[ei + 1].wg_begin <= (int)blockIdx.x) ++ei;
  const RepEp E = batch.e[ei];
  const int local = (int)blockIdx.x - E.wg_begin;
  const int pair = local / E.parts, part = local % E.parts;
  const int64_t ct = E.text0 + E.ntexts - 1, bt = E.text0 + pair;
  const int64_t a0 = toff[ct], a1 = toff[ct + 1], b0 = toff[bt], b1 = toff[bt + 1];

  extern __shared__ __align__(16) uint8_t smem[];
  uint32_t* ta = reinterpret_cast<uint32_t*>(smem);  // [kRepSlots] candidate words of the partition
  uint32_t* tb = ta + kRepSlots;                     // [kRepSlots] previous text's words
  __shared__ int cnt[4];                             // |A|, |B|, |A & B|, full
  const int tid = threadIdx.x;
  {
    u32x4* t4 = reinterpret_cast<u32x4*>(smem);
    for (int i = tid; i < 2 * kRepSlots / 4; i += 1024) t4[i] = u32x4{kRepEmpty, kRepEmpty, kRepEmpty, kRepEmpty};
    if (tid < 4) cnt[tid] = 0;
  }
  __syncthreads();
  int na = 0, full = 0;
  for (int64_t i = a0 + tid; i < a1; i += 1024) {
    const int32_t w = words[i];
    const uint32_t h = word_hash(w);
    if (part_of(h, E.parts) != part) continue;
    const int r = set_insert(ta, h, (uint32_t)w);
    na += r > 0;
    full |= r < 0;
  }
  __syncthreads();
  int nb = 0, ni = 0;
  for (int64_t i = b0 + tid; i < b1; i += 1024) {
    const int32_t w = words[i];
    const uint32_t h = word_hash(w);
    if (part_of(h, E.parts) != part) continue;
    const int r = set_insert(tb, h, (uint32_t)w);
    if (r > 0) {
      ++nb;
      ni += set_contains(ta, h, (uint32_t)w);
    }
    full |= r < 0;
  }
  // per-thread counts, then one LDS atomic each
  if (na) atomicAdd(cnt + 0, na);
  if (nb) atomicAdd(cnt + 1, nb);
  if (ni) atomicAdd(cnt + 2, ni);
  if (full) atomicOr(cnt + 3, 1);
  __syncthreads();
  if (tid < 4) counts[(E.wg_global + local) * 4 + tid] = cnt[tid];
}

__global__ __launch_bounds__(64) void rep_reduce_kernel(RepBatch batch, const int32_t* __restrict__ counts, double tau,
                                                        double* __restrict__ rho, double* __restrict__ nu,
                                                        int32_t* __restrict__ skip, int32_t* __restrict__ best,
                                                        int32_t* __restrict__ pair_counts) {
  const int ei = (int)threadIdx.x;
  if (ei >= batch.count) return;
  const RepEp E = batch.e[ei];
  int64_t bi = 1, bu = 1;  // best fraction bi / bu, starting below every J (0 / 1 is attained)
  int bk = -1;
  bool bad = false;
  for (int k = 0; k + 1 < E.ntexts; ++k) {
    int64_t a = 0, b = 0, in = 0;
    for (int p = 0; p < E.parts; ++p) {
      const int32_t* c = counts + (E.wg_global + (int64_t)k * E.parts + p) * 4;
      a += c[0];
      b += c[1];
      in += c[2];
      bad |= c[3] != 0;
    }
    const int64_t un = a + b - in;
    if (pair_counts) {
      pair_counts[(E.pair_base + k) * 2] = (int32_t)in;
      pair_counts[(E.pair_base + k) * 2 + 1] = (int32_t)un;
    }
    // J = in / un (0 when un = 0); J > best  <=>  in * bu > bi * un (the first maximum stays)
    const int64_t ju = un > 0 ? un : 1;
    if (bk < 0 || in * bu > bi * ju) {
      bk = k;
      bi = in;
      bu = ju;
    }
  }
  double r = 0.0;
  if (bk >= 0) r = __ddiv_rn((double)bi, (double)bu);
  const double v = __dsub_rn(1.0, r);
  const int e = E.ep;
  if (bad) {
    rho[e] = __longlong_as_double(0x7FF8000000000000ll);
    nu[e] = __longlong_as_double(0x7FF8000000000000ll);
    skip[e] = 0;
    best[e] = -1;
    return;
  }
  rho[e] = r;
  nu[e] = v;
  skip[e] = v < tau ? 1 : 0;
  best[e] = bk;
}

hipError_t launch_rep_count(const RepBatch& b, int total_wgs, const int32_t* words, const int64_t* toff,
                            int32_t* counts, hipStream_t s) {
  if (total_wgs <= 0) return hipSuccess;
  static bool attr = false;
  const size_t lds = (size_t)2 * kRepSlots * 4;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)rep_count_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  KernelTimer t(K_REP_COUNT, s);
  hipLaunchKernelGGL(rep_count_kernel, dim3(total_wgs), dim3(1024), lds, s, b, words, toff, counts);
  return hipGetLastError();
}

hipError_t launch_rep_reduce(const RepBatch& b, const int32_t* counts, double tau, double* rho, double* nu,
                             int32_t* skip, int32_t* best, int32_t* pair_counts, hipStream_t s) {
  if (b.count <= 0) return hipSuccess;
  KernelTimer t(K_REP_REDUCE, s);
  hipLaunchKernelGGL(rep_reduce_kernel, dim3(1), dim3(64), 0, s, b, counts, tau, rho, nu, skip, best, pair_counts);
  return hipGetLastError();
}

}  // namespace attt
