// bf16 backward of the token-weighted CE (the gradient of Eq. 10 with respect to the hidden
// states) in one persistent kernel: no buffer of (rows x vocabulary) ever exists in memory.
//
// dL/dh_t = (w_t / L_e) (softmax(z_t) - onehot(y_t)) W is a contraction over the vocabulary of a
// per-row gradient tile with W. The kernel splits that into two roles that run concurrently on the
// 32 CUs of each XCD:
//   producers  compute a 256 (vocab) x 256 (token) logit tile z^T = W h^T on MFMA, turn it into
//              the tile's share of the gradient (label mode: e = exp(z - z_y) off the label, the
//              softmax numerators referenced to the label logit; exact mode: coef p with
//              p = exp(z - lse), for rows with p_y > 1/2 coef (p - onehot(y)), the label entry's
//              p_y - 1 formed in float32) in bf16, and publish it into a slot of a small ring that
//              stays in the XCD's L2;
//   consumers  own one 256-column slice of d for a 256-row tile and accumulate
//              acc (+)= W^T[slice, vocab tile] * tile^T in float32 registers over the whole
//              vocabulary, reading the ring, then write dL/dh = sa acc - sb W_y (label mode:
//              sa = coef / (1 + sigma), sb = sigma sa, sigma from the producers' per-tile sums,
//              the label term applied in float32 from W; exact mode: sa = 1, sb = coef, or 0 for
//              rows whose label term is in the tile). Neither mode rounds a value near coef (the
//              label entry's p_y of a confident row) to bf16 and subtracts the label term
//              afterwards: that would leave (1 - p_y) with the absolute error of bf16 at 1.
// Teams form at run time: every workgroup reads the id of the XCD it runs on, takes a rank in that
// XCD's team by an atomic counter, and after a grid barrier all workgroups check that every team
// has exactly kTeam members. Team x works on the row tiles x, x + 8, x + 16, ...; a ring slot is
// written and read only by workgroups of one XCD, i.e. through one L2.
//
// Signalling. Flags are agent-scope atomics on a zeroed sync area (relaxed loads and stores are
// performed at the memory side on gfx950, read-modify-write atomics are device-coherent), with no
// release / acquire fences, which would write back or invalidate the whole L2. The data a flag
// announces is written with ordinary stores, waited for with s_waitcnt (the L2 has acknowledged
// them) before the flag is set, and read by the same XCD with loads that bypass the CU's L1 (sc0).
//   published[item] 1 once the item's tile is in its slot, set by its producer;
//   consumed[slot]  +1 from each of a consumer's four loading waves once its loads of the slot have
//                   landed; a producer reuses a slot when all consumers have signalled its last use.
// Every wait is bounded by a wall-clock limit: a wait that runs out raises the abort flag, every
// later wait returns at once, and workgroups skip their remaining work at the next item, so every
// wave exits. Control flow is uniform within a workgroup around every barrier (abort decisions go
// through LDS). An abort (or an overflow of the label-referenced sums) raises the caller's guard
// flag, on which the exact path reruns.
#include "common.hpp"
#include "gemm_core.hpp"
#include "internal.hpp"

namespace attt {

constexpr int kSlotBytes = 256 * 256 * 2;  // one bf16 tile [256 tokens][256 vocab]
// Dynamic LDS: the mainloops' two stage buffers and group counter (CfgBig::LDS), the producer's
// per-token sums [2][256], then four ints of workgroup state. There is no static LDS, so the
// stage buffers start at LDS address 0.
constexpr size_t kFusedLdsData = CfgBig::LDS + 2 * 256 * sizeof(float);
constexpr size_t kFusedLds = kFusedLdsData + 4 * sizeof(int);

// sync area (ints): team counts [8], arrive, abort, the site of the first wait that ran out
// (diagnostics: 1 grid barrier, 2 consumer awaiting a tile, 3 producer awaiting a free slot,
// 4 idle consumer, 5 partial sums of the vocabulary split), then consumed [8][S] per ring slot,
// published [8][G] per item (G: the most items a team has, a multiple of 4) and, per team, the
// split's ready [kCeTeam] and freed [kCeTeam] counters
constexpr int kSyncTeam = 0, kSyncArrive = 8, kSyncAbort = 9, kSyncSite = 10, kSyncSlots = 16;
enum { kSiteGrid = 1, kSiteTile = 2, kSiteSlot = 3, kSiteIdle = 4, kSitePartial = 5 };

__device__ __forceinline__ int ld_agent(const int* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int add_agent(int* p, int v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until *p >= target; false if the abort flag is (or gets) raised. After `limit` ticks of
// the 100 MHz wall clock without success it raises the abort flag itself. p is wave-uniform.
// `abort` is the sync area's abort flag; the int after it records the site of a wait that ran out.
__device__ __forceinline__ bool wait_geq(const int* p, int target, int* abort, uint64_t limit, int site) {
  if (ld_agent(p) >= target) return true;
  const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
  while (true) {
    if (ld_agent(abort) != 0) return false;
    if (ld_agent(p) >= target) return true;
    if (__builtin_amdgcn_s_memrealtime() - t0 > limit) {
      int none = 0;
      __hip_atomic_compare_exchange_strong(abort + (kSyncSite - kSyncAbort), &none, site, __ATOMIC_RELAXED,
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      st_agent(abort, 1);
      return false;
    }
    __builtin_amdgcn_s_sleep(2);
  }
}

// Acquire side of a flag: after the flag has been observed, invalidate this CU's L1 so that no
// later load of the data the flag announces can be served by a stale L1 line (the L2 holds the
// data; the same sequence as a workgroup-scope acquire on gfx950: sc0 load, then buffer_inv sc0).
__device__ __forceinline__ void l1_invalidate() { asm volatile("buffer_inv sc0" ::: "memory"); }

// Waits as wait_geq and then invalidates the CU's L1 (the acquire of the announced data).
__device__ __forceinline__ bool acquire_geq(const int* p, int target, int* abort, uint64_t limit, int site);

// id of the XCD this wave runs on (hardware register XCC_ID, bits 3:0)
__device__ __forceinline__ int xcc_id() { return __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 7; }

__device__ __forceinline__ bool acquire_geq(const int* p, int target, int* abort, uint64_t limit, int site) {
  const bool ok = wait_geq(p, target, abort, limit, site);
  l1_invalidate();
  return ok;
}

// Exact mode, where the label term -coef W_y of a row goes. Folded into the tile entry
// coef (p_y - 1) (formed in float32, then rounded to bf16) its error is 2^-9 coef (1 - p_y) |W_y|;
// kept out (the entry is coef p_y, the consumer subtracts coef W_y in float32) it is
// 2^-9 coef p_y |W_y|. Fold when p_y = exp(z_y - lse) > 1/2. Producer and consumer take the
// decision from the same stored z_y and lse, so they always agree.
__device__ __forceinline__ bool exact_fold(float z_y, float lse) { return z_y - lse > -0.69314718f; }

// The consumer's GEMM: acc += A[0:256, 0:K] T^T with T the ring tiles of items gbase,
// gbase + step, ..., nitems of them, laid end to end along K (each [256 tokens][256 vocab]);
// A = W^T rows of the d-slice, read at the items' vocabulary columns (item i is vocabulary tile
// vfirst + i step). The same 8-wave ping-pong as mfma_mainloop_pp16, with the same group counter before
// group 1's refills; only group 1 (waves 4-7) loads ring blocks inside the loop (group 0's share
// of a stage is A blocks), so group 1 waits for an item's ready flag before issuing its first
// stage (ensure: flags read 16 items at a time), and signals `consumed` once its loads of the
// item's last stage have landed. The prologue (group 0 issues all of stage 0) waits for item
// gbase in every wave.
template <class C>
__device__ __forceinline__ void consumer_mainloop(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                                  const uint8_t* ring, int nval, int nitems, int gbase, int step,
                                                  int vfirst, int S, const int* published, int* consumed, int* abort,
                                                  uint64_t limit, bf16_t* lds, Acc16& acc, int tid) {
  static_assert(C::NT == 512 && C::WGM == 2 && C::WGN == 4 && C::BN == 256, "8 waves over 256-token tiles");
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int grp = wave >> 2;
#pragma unroll
  for (int i = 0; i < Mma16::TM; ++i)
#pragma unroll
    for (int j = 0; j < Mma16::TN; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  const __amdgpu_buffer_rsrc_t rA = make_rsrc(A);
  const __amdgpu_buffer_rsrc_t rR = buffer_rsrc(ring, S * kSlotBytes);
  constexpr int LW = 4;
  constexpr int ABLK = C::BM / 8;
  constexpr int BPW = (ABLK + C::BN / 8) / LW;
  // Group 0 loads blocks [kCs, kCs + 6) of each stage, A rows only (the ring rows are loaded by
  // group 1, which waits for their flags); group 1 loads [0, kCs), A rows of group 0's half
  // that no wave of group 1 reads, then the ring rows [JA, BPW) once all four of its waves have
  // read the stage (see PpLoader in gemm_core.hpp).
  constexpr int kCs = 2;
  static_assert(kCs + 6 == ABLK / LW && kCs * LW * 8 <= C::WTM, "group 0's share holds A blocks only");
  const int lr = lane >> 3;
  const int c_even = (lane & 7) ^ ((lr >> 1) & 7);
  const int c_odd = (lane & 7) ^ (((8 + lr) >> 1) & 7);
  const uint32_t la = (uint32_t)(lr * lda * 2);
  const int nk = 4 * nitems;
  // blocks j < JA of a stage are A rows (W^T), the rest ring rows
  constexpr int JA = ABLK / LW;
  auto dma = [&](int st, int k, int j0, int j1) {
    bf16_t* base = lds + st * (C::SA + C::SB);
    const int slot = (gbase + (k >> 2) * step) % S;
    const uint32_t kcol = (uint32_t)(k & 3) * 64;
    // the stage's vocabulary columns: item k / 4 is vocabulary tile vfirst + (k / 4) step
    const int vcol = (vfirst + (k >> 2) * step) * 256 + (int)kcol;
#pragma unroll
    for (int j = j0; j < j1 && j < JA; ++j) {
      const int blk = (wave & 3) + j * LW;
      const int rb = blk * 8;
      const int c = (rb & 8) ? c_odd : c_even;
      const bool ok = rb + lr < mval;
      const uint32_t off = (uint32_t)((int64_t)rb * lda * 2) + la + (uint32_t)(vcol + c * 8) * 2;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rA, (__attribute__((address_space(3))) void*)(base + blk * 512), 16,
                                               ok ? off : kOOB, 0, 0, 0);
    }
#pragma unroll
    for (int j = j0 > JA ? j0 : JA; j < j1; ++j) {
      const int blk = (wave & 3) + j * LW;
      const int rb = (blk - ABLK) * 8;
      const int c = (rb & 8) ? c_odd : c_even;
      const bool ok = rb + lr < nval;
      const uint32_t off = (uint32_t)slot * kSlotBytes + (uint32_t)(rb + lr) * 512 + (kcol + c * 8) * 2;
      // ring rows bypass the CU's L1 (sc0): the slot was rewritten since this CU last read it
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rR, (__attribute__((address_space(3))) void*)(base + blk * 512), 16,
                                               ok ? off : kOOB, 0, 0, 1);
    }
  };
  bf16x8 fa[2][Mma16::TM], fb[2][Mma16::TN];
  auto mem = [&](int k) {
    const bf16_t* As = lds + (k & 1) * (C::SA + C::SB);
    mma16_frags<C>(As, As + C::SA, lane, wm, wn, fa, fb);
  };
  auto compute = [&]() { mma16_step(fa, fb, acc); };
  auto pin = [&]() { mma16_pin(acc); };
  auto slot_of = [&](int item) { return (gbase + item * step) % S; };
  // Items [0, known) of this mainloop are known to be published. ensure(i) makes item i known:
  // one 16-byte memory-side load (sc1, as a relaxed agent-scope atomic load is) reads the
  // published flags of the four items of its aligned group, and every consecutive published item
  // from i on becomes known, so while the producers run ahead the flags cost one round trip per
  // four items. New items are acquired with an L1 invalidate. The wait is bounded like wait_geq.
  const __amdgpu_buffer_rsrc_t rP = buffer_rsrc(published, ((gbase + (nitems - 1) * step) / 4 + 1) * 16);
  int known = 0;
  auto ensure = [&](int i) {
    if (i < known) return;
    const int g = gbase + i * step, g4 = g & ~3;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (true) {
      const u32x4 fv = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rP, (uint32_t)g4 * 4u, 0, 16));
      // every lane read the same four flags: keep them (and what follows from them) scalar
      const uint32_t f[4] = {(uint32_t)__builtin_amdgcn_readfirstlane(fv[0]), (uint32_t)__builtin_amdgcn_readfirstlane(fv[1]),
                             (uint32_t)__builtin_amdgcn_readfirstlane(fv[2]), (uint32_t)__builtin_amdgcn_readfirstlane(fv[3])};
      int j = g - g4, run = 0;
      while (j < 4 && f[j] != 0u) j += step, ++run;
      if (run > 0) {
        known = i + run;
        l1_invalidate();
        return;
      }
      if (ld_agent(abort) != 0) break;
      if (__builtin_amdgcn_s_memrealtime() - t0 > limit) {
        int none = 0;
        __hip_atomic_compare_exchange_strong(abort + (kSyncSite - kSyncAbort), &none, (int)kSiteTile,
                                             __ATOMIC_RELAXED, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        st_agent(abort, 1);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    known = i + 1;  // aborted: go on with whatever the slot holds, the result is discarded
  };
  const uint32_t ctr = group1_counter<C>(lds);
  group1_reset(ctr, tid);
  ensure(0);
  if (grp == 0) dma(0, 0, 0, BPW);
  __builtin_amdgcn_s_waitcnt(0);
  if (grp == 1 && nk > 1) {
    dma(1, 1, 0, kCs);
    dma(1, 1, JA, BPW);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the counter reset has landed
  wg_barrier();
  if (grp == 0) {
    for (int k = 0; k < nk; ++k) {
      if (k + 1 < nk) dma((k + 1) & 1, k + 1, kCs, JA);
      mem(k);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();
      pin();
      compute();
      pin();
      __builtin_amdgcn_s_waitcnt(0);
      wg_barrier();
    }
    wg_barrier();
  } else {
    wg_barrier();
    for (int k = 0; k < nk; ++k) {
      mem(k);
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      // stage k+1 (issued last iteration) has landed: at k = 4i + 2 that is item i's last stage
      if ((k & 3) == 2 && __builtin_amdgcn_mbcnt_lo(~0u, 0u) == 0) add_agent(consumed + slot_of(k >> 2), 1);
      if (k + 2 < nk) {
        if (((k + 2) & 3) == 0) ensure((k + 2) >> 2);
        group1_arrive(ctr, lane);
        dma(k & 1, k + 2, 0, kCs);
        // the other waves of group 1 read the ring rows this refill overwrites
        group1_wait(ctr, k);
        dma(k & 1, k + 2, JA, BPW);
      }
      wg_barrier();
      pin();
      compute();
      pin();
      wg_barrier();
    }
  }
}

// The kernel body. kSplit: the consumers split the vocabulary tiles of a d-slice (F = ksplit > 1);
// a separate instantiation, so that the kernel without it keeps its own register allocation.
template <bool kLabel, bool kSplit>
__device__ __forceinline__ void ce_fused_body(const CeFusedArgs& a) {
  using C = CfgBig;
  extern __shared__ __align__(16) uint8_t smem[];
  int* info = reinterpret_cast<int*>(smem + kFusedLdsData);
  int* sync = a.sync;
  int* abort = sync + kSyncAbort;
  const int tid = threadIdx.x;
  // the exact mode runs only when the label-referenced pass raised the guard flag
  if (!kLabel && *a.gate == 0) return;

  // ---- team formation ----
  if (tid == 0) {
    const int x = xcc_id();
    const int rank = add_agent(sync + kSyncTeam + x, 1);
    __builtin_amdgcn_s_waitcnt(0);  // the team count has been taken before arrival is announced
    add_agent(sync + kSyncArrive, 1);
    bool ok = wait_geq(sync + kSyncArrive, (int)gridDim.x, abort, a.limit, kSiteGrid);
    for (int i = 0; ok && i < 8; ++i) ok = ld_agent(sync + kSyncTeam + i) == kCeTeam;
    if (!ok) st_agent(abort, 1);
    info[0] = x;
    info[1] = rank;
    info[2] = ok ? 1 : 0;
  }
  __syncthreads();
  if (!__builtin_amdgcn_readfirstlane(info[2])) return;
  const int x = __builtin_amdgcn_readfirstlane(info[0]), rank = __builtin_amdgcn_readfirstlane(info[1]);
  const int P = kCeTeam - a.consumers, Cn = a.consumers;
  const int nrt = x < a.row_tiles ? (a.row_tiles - x + 7) / 8 : 0;  // row tiles of this team
  const int per_tile = a.passes * a.nv;                              // items per row tile
  const int items = nrt * per_tile;
  const int S = a.slots;
  uint8_t* ring = a.ring + (size_t)x * S * kSlotBytes;
  int* consumed = sync + kSyncSlots + x * S;
  int* published = sync + kSyncSlots + 8 * S + x * a.items_max;
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);

  if (rank < P) {
    // ---- producer: items rank, rank + P, ... ----
    for (int g = rank; g < items; g += P) {
      if (tid == 0) info[3] = ld_agent(abort);
      __syncthreads();
      if (__builtin_amdgcn_readfirstlane(info[3])) break;
      // the thread index, opaque to the compiler inside the loop: the per-lane offsets below are
      // recomputed per item instead of being held in registers across the mainloop
      int tix = tid;
      asm volatile("" : "+v"(tix));
      const int lane = tix & 63, wave = __builtin_amdgcn_readfirstlane(tix >> 6);
      const int wm = wave / C::WGN, wn = wave % C::WGN;
      const int j = g / per_tile, rem = g % per_tile;
      const int pass = rem / a.nv, v = rem % a.nv;
      const int t0 = (x + 8 * j) * 256, v0 = v * 256;
      const int R = min(256, a.N - t0);
      const int slot = g % S;
      Acc16 acc;
      // the first stages of every item after the first were issued during the previous epilogue
      mfma_mainloop_pp16<C>(a.W + (int64_t)v0 * a.d, a.d, a.V - v0, a.h + (int64_t)t0 * a.d, a.d, R, a.d, lds, acc,
                          tix, g != rank);
      // the slot's previous use must have been read by every consumer (four waves each)
      // (four waves of every consumer that reads the slot: all of them with one consumer per
      // d-slice, whose idle ones pace too; with the vocabulary split, one per d-slice)
      wait_geq(consumed + slot, 4 * (kSplit ? a.slices : Cn) * (g / S), abort, a.limit, kSiteSlot);
      // start the next item's first stages now, so that their latency hides behind this epilogue
      // (they land before the publish below; an abort at the next item's check finds them landed)
      if (g + P < items) {
        const int gn = g + P, jn = gn / per_tile, vn = gn % per_tile % a.nv;
        const int t0n = (x + 8 * jn) * 256, v0n = vn * 256;
        mfma_pp_prologue<C>(a.W + (int64_t)v0n * a.d, a.d, a.V - v0n, a.h + (int64_t)t0n * a.d, a.d,
                            min(256, a.N - t0n), a.d, lds, tix);
      }
      bf16_t* tile = reinterpret_cast<bf16_t*>(ring + (size_t)slot * kSlotBytes);
      // [WGM][256] per-token sums of the tile, after the two stage buffers (which hold the next
      // item's first stages by now)
      float* red = reinterpret_cast<float*>(smem + C::LDS);
      const int vb = v0 + wm * C::WTM;
      const bool full = v0 + C::BM <= a.V;
      constexpr float kLog2e = 1.4426950408889634f;
      constexpr float kOverSum = 6.2351491e27f;  // e^64
      const int q4 = lane >> 4;
      bool over = false;
#pragma unroll
      for (int jj = 0; jj < Mma16::TN; ++jj) {
        const int tl = wn * C::WTN + jj * 16 + Mma16::col(lane);
        const bool tok = tl < R;
        float ref = 0.0f, cf = 0.0f;
        int y = -1;
        bool fold = false;  // exact mode: the label term goes into the tile (see exact_fold)
        if (tok) {
          y = a.labels[t0 + tl];
          ref = kLabel ? a.label_logit[t0 + tl] : a.lse[t0 + tl];
          cf = kLabel ? 0.0f : a.coef[t0 + tl];
          if (!kLabel) fold = exact_fold(a.label_logit[t0 + tl], ref);
        }
        const float nref = -ref * kLog2e;
        const int ylane = y - vb - 4 * q4;  // the label's offset from this lane's first vocab row
        // exact mode, label outside [0, V) (outside the contract): NaN gradient row
        const bool bad = !kLabel && tok && (y < 0 || y >= a.V);
        if (bad) cf = __int_as_float(0x7FC00000);
        float sum = 0.0f;
#pragma unroll
        for (int i = 0; i < Mma16::TM; i += 2) {
          uint32_t pk[2][2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int yl = ylane - (i + h) * 16;
            float e[4];
            if (!full || __ballot(yl >= 0 && yl < 4) != 0) {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int vv = vb + (i + h) * 16 + Mma16::row(r, lane);
                const float ex = __builtin_amdgcn_exp2f(fmaf(acc[i + h][jj][r], kLog2e, nref));
                if (kLabel) e[r] = (vv < a.V && vv != y) ? ex : 0.0f;
                else e[r] = vv < a.V ? cf * ((fold && vv == y) ? ex - 1.0f : ex) : 0.0f;
              }
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const float ex = __builtin_amdgcn_exp2f(fmaf(acc[i + h][jj][r], kLog2e, nref));
                e[r] = kLabel ? ex : cf * ex;
              }
            }
            sum += e[0];
            sum += e[1];
            sum += e[2];
            sum += e[3];
            pk[h][0] = pack_bf16x2(e[0], e[1]);
            pk[h][1] = pack_bf16x2(e[2], e[3]);
          }
          // Lane row q4 holds vocab 4 q4 .. 4 q4 + 3 of tiles i and i + 1. Swapping the odd
          // 16-lane rows of tile i's words with the even rows of tile i + 1's leaves every even-row
          // lane with 8 consecutive vocab entries of tile i (its own four, then those of the lane
          // 16 above) and every odd-row lane with 8 of tile i + 1: one 16-byte store each.
          uint32_t w[4];
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const auto sw = __builtin_amdgcn_permlane16_swap(pk[0][k], pk[1][k], false, false);
            w[k] = sw[0];
            w[2 + k] = sw[1];
          }
          if (tok) {
            const int odd = q4 & 1;
            const int voff = (vb - v0) + (i + odd) * 16 + 4 * (q4 - odd);
            *reinterpret_cast<u32x4*>(tile + tl * 256 + voff) = u32x4{w[0], w[1], w[2], w[3]};
          }
        }
        if (kLabel) {
          over |= sum > kOverSum;
          sum += __shfl_xor(sum, 16, 64);
          sum += __shfl_xor(sum, 32, 64);
          if (q4 == 0) red[wm * C::BN + tl] = sum;
        }
      }
      if (kLabel) {
        if (over) *a.gate = 1;
        __syncthreads();
        if (pass == 0)
          for (int tl = tix; tl < R; tl += C::NT) {
            float sum = red[tl];
#pragma unroll
            for (int w = 1; w < C::WGM; ++w) sum += red[w * C::BN + tl];
            a.sig_part[(int64_t)(t0 + tl) * a.nv + v] = sum;
          }
      }
      __builtin_amdgcn_s_waitcnt(0);  // this wave's stores of the tile (and sums) are in the L2
      __syncthreads();
      if (tix == 0) st_agent(published + g, 1);
    }
    return;
  }

  // ---- consumer: a d-slice of every row tile of the team, items in order ----
  const int c = rank - P;
  for (int j = 0; j < nrt; ++j) {
    const int t0 = (x + 8 * j) * 256;
    const int R = min(256, a.N - t0);
    for (int pass = 0; pass < a.passes; ++pass) {
      if (tid == 0) info[3] = ld_agent(abort);
      __syncthreads();
      if (__builtin_amdgcn_readfirstlane(info[3])) return;
      int tix = tid;  // opaque inside the loop, as in the producer
      asm volatile("" : "+v"(tix));
      const int lane = tix & 63, wave = __builtin_amdgcn_readfirstlane(tix >> 6);
      const int wm = wave / C::WGN, wn = wave % C::WGN;
      const int gbase = (j * a.passes + pass) * a.nv;
      // with the vocabulary split (F = ksplit > 1, one pass), consumer c takes d-slice c % slices
      // and, as part c / slices, the vocabulary tiles part, part + F, ...
      const int F = kSplit ? a.ksplit : 1;
      const int slice = kSplit ? c % a.slices : pass * Cn + c;
      const int part = kSplit ? c / a.slices : 0;
      if (!kSplit && slice >= a.slices) {
        // idle in this pass, but every consumer paces and releases every slot
        if (wave >= 4)
          for (int v = 0; v < a.nv; ++v) {
            wait_geq(published + gbase + v, 1, abort, a.limit, kSiteIdle);
            if (lane == 0) add_agent(consumed + (gbase + v) % S, 1);
          }
        continue;
      }
      const int m0 = slice * 256;  // first column of dL/dh
      Acc16 acc;
      consumer_mainloop<C>(a.WT + (int64_t)m0 * a.Vp, a.Vp, a.d - m0, ring, R, (a.nv - part + F - 1) / F,
                           gbase + part, F, part, S, published, consumed, abort, a.limit, lds, acc, tix);
      if constexpr (kSplit) {
        // Parts 1 .. F-1 hand their float32 sums to part 0 through a per-(team, slice, part)
        // buffer, in the thread order of the accumulators; part 0 adds them in part order (a
        // fixed order) and writes the slice. Flags (per team): ready[c] = row tiles whose sums
        // consumer c has written, freed[slice] = row tiles whose sums part 0 has read.
        int* ready = sync + kSyncSlots + 8 * S + 8 * a.items_max + x * 2 * kCeTeam;
        int* freed = ready + kCeTeam;
        const size_t per = (size_t)256 * 256;
        float* mine = a.partial + (((size_t)x * a.slices + slice) * (F - 1)) * per;
        if (part > 0) {
          float* dst = mine + (size_t)(part - 1) * per;
          wait_geq(freed + slice, j, abort, a.limit, kSitePartial);  // row tile j-1's sums were read
#pragma unroll
          for (int i = 0; i < Mma16::TM; ++i)
#pragma unroll
            for (int jj = 0; jj < Mma16::TN; ++jj)
              *reinterpret_cast<f32x4*>(dst + ((size_t)(i * Mma16::TN + jj) * C::NT + tix) * 4) = acc[i][jj];
          __builtin_amdgcn_s_waitcnt(0);  // this wave's sums are in the L2
          __syncthreads();
          if (tix == 0) st_agent(ready + c, j + 1);
          continue;  // part 0 writes the slice
        }
        for (int f = 1; f < F; ++f) {
          wait_geq(ready + f * a.slices + slice, j + 1, abort, a.limit, kSitePartial);
          l1_invalidate();
          const float* src = mine + (size_t)(f - 1) * per;
#pragma unroll
          for (int i = 0; i < Mma16::TM; ++i)
#pragma unroll
            for (int jj = 0; jj < Mma16::TN; ++jj) {
              const f32x4 v = *reinterpret_cast<const f32x4*>(src + ((size_t)(i * Mma16::TN + jj) * C::NT + tix) * 4);
#pragma unroll
              for (int e = 0; e < 4; ++e) acc[i][jj][e] += v[e];
            }
        }
        __syncthreads();  // every wave has its sums of all parts
        if (tix == 0) st_agent(freed + slice, j + 1);
      }
      // row scales: sigma_t from the producers' per-tile sums in a fixed order (two threads per
      // token: even and odd vocab tiles), sa = coef / (1 + sigma), sb = coef sigma / (1 + sigma)
      float* sig = reinterpret_cast<float*>(smem);  // [256][2], after the mainloop's last barrier
      if (kLabel) {
        l1_invalidate();  // the sums were published with the ready flags this workgroup observed
        const int tl = tix >> 1, half = tix & 1;
        // one descriptor over the row tile's sums (its base must be uniform), per-lane offsets
        const __amdgpu_buffer_rsrc_t rp = buffer_rsrc(a.sig_part + (int64_t)t0 * a.nv, R * a.nv * 4);
        float s = 0.0f;
        if (tl < R) {
          const uint32_t row_off = (uint32_t)(tl * a.nv) * 4u;
#pragma unroll 8
          for (int v = half; v < a.nv; v += 2)
            s += __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rp, row_off + v * 4, 0, 1));
        }
        sig[tix] = s;
        __syncthreads();
      }
      const int q4 = lane >> 4;
#pragma unroll
      for (int jj = 0; jj < Mma16::TN; ++jj) {
        const int tl = wn * C::WTN + jj * 16 + Mma16::col(lane);
        const bool tok = tl < R;
        float sa = 1.0f, sb = 0.0f;
        const bf16_t* wy = nullptr;
        if (tok) {
          const int row = t0 + tl;
          const float cf = a.coef[row];
          if (kLabel) {
            const float sigma = sig[2 * tl] + sig[2 * tl + 1];
            const float inv = __fdiv_rn(1.0f, 1.0f + sigma);
            sa = cf * inv;
            sb = cf * (sigma * inv);
          } else if (!exact_fold(a.label_logit[row], a.lse[row])) {
            sb = cf;  // the label term in float32; a folded one is inside acc already
          }
          const int y = a.labels[row];
          if (y < 0 || y >= a.V) sa = __int_as_float(0x7FC00000);  // outside the contract: NaN row
          else if (sb != 0.0f) wy = a.W + (int64_t)y * a.d;
        }
#pragma unroll
        for (int i = 0; i < Mma16::TM; i += 2) {
          uint32_t pk[2][2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            // this lane's four columns of d in tile i + h
            const int cc = m0 + wm * C::WTM + (i + h) * 16 + Mma16::row(0, lane);
            float wv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            if (wy && cc + 4 <= a.d) {
              const uint2 u = *reinterpret_cast<const uint2*>(wy + cc);
              wv[0] = bf16_bits_to_f32(u.x & 0xFFFFu);
              wv[1] = bf16_bits_to_f32(u.x >> 16);
              wv[2] = bf16_bits_to_f32(u.y & 0xFFFFu);
              wv[3] = bf16_bits_to_f32(u.y >> 16);
            }
            float vv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) vv[e] = sa * acc[i + h][jj][e] - sb * wv[e];
            pk[h][0] = pack_bf16x2(vv[0], vv[1]);
            pk[h][1] = pack_bf16x2(vv[2], vv[3]);
          }
          // as in the producer: even-row lanes end up with 8 consecutive columns of tile i,
          // odd-row lanes with 8 of tile i + 1
          uint32_t w[4];
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const auto sw = __builtin_amdgcn_permlane16_swap(pk[0][k], pk[1][k], false, false);
            w[k] = sw[0];
            w[2 + k] = sw[1];
          }
          const int odd = q4 & 1;
          const int c8 = m0 + wm * C::WTM + (i + odd) * 16 + 4 * (q4 - odd);
          if (tok && c8 + 8 <= a.d)
            *reinterpret_cast<u32x4*>(a.grad + (int64_t)(t0 + tl) * a.d + c8) = u32x4{w[0], w[1], w[2], w[3]};
        }
      }
      __syncthreads();  // sig and the mainloop's LDS are reused by the next pass
    }
  }
}

template <bool kLabel>
__global__ __launch_bounds__(512) void ce_fused_bwd_kernel(CeFusedArgs a) {
  ce_fused_body<kLabel, false>(a);
}
template <bool kLabel>
__global__ __launch_bounds__(512) void ce_fused_bwd_split_kernel(CeFusedArgs a) {
  ce_fused_body<kLabel, true>(a);
}

// Zeroes `n` ints (the sync areas) with vector stores.
__global__ __launch_bounds__(256) void ce_sync_clear_kernel(int* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

// After the label-referenced pass: an aborted pass raises the guard flag.
__global__ void ce_fused_status_kernel(const int* sync, int* gate) {
  if (threadIdx.x == 0 && sync[kSyncAbort] != 0) *gate = 1;
}

// After the exact pass: if it aborted too, every output is NaN (no result is trusted).
__global__ __launch_bounds__(256) void ce_fused_nan_kernel(const int* sync, float* loss, int E, float* lse, int N,
                                                           bf16_t* grad, int64_t nd) {
  if (sync[kSyncAbort] == 0) return;
  const int64_t stride = (int64_t)gridDim.x * 256;
  const int64_t i0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (int64_t i = i0; i < nd; i += stride) grad[i] = (bf16_t)0x7FC0;
  for (int64_t i = i0; i < N; i += stride) lse[i] = __int_as_float(0x7FC00000);
  for (int64_t i = i0; i < E; i += stride) loss[i] = __int_as_float(0x7FC00000);
}

// ------------------------------------------------------------------------------------------
size_t ce_fused_ring_bytes(int slots) { return (size_t)8 * slots * kSlotBytes; }
int ce_fused_sync_ints(int slots, int items_max) {
  return kSyncSlots + 8 * slots + 8 * items_max + 8 * 2 * kCeTeam;
}

hipError_t launch_ce_sync_clear(int* sync, int n, hipStream_t s) {
  const int blocks = (n + 255) / 256 < 64 ? (n + 255) / 256 : 64;
  hipLaunchKernelGGL(ce_sync_clear_kernel, dim3(blocks), dim3(256), 0, s, sync, n);
  return hipGetLastError();
}

hipError_t launch_ce_fused(bool label, const CeFusedArgs& a, hipStream_t s) {
  const void* fns[2][2] = {{reinterpret_cast<const void*>(ce_fused_bwd_kernel<false>),
                            reinterpret_cast<const void*>(ce_fused_bwd_split_kernel<false>)},
                           {reinterpret_cast<const void*>(ce_fused_bwd_kernel<true>),
                            reinterpret_cast<const void*>(ce_fused_bwd_split_kernel<true>)}};
  static bool attr = false;
  if (!attr) {
    for (int i = 0; i < 4; ++i) {
      hipError_t e = hipFuncSetAttribute(fns[i >> 1][i & 1], hipFuncAttributeMaxDynamicSharedMemorySize, (int)kFusedLds);
      if (e != hipSuccess) return e;
    }
    attr = true;
  }
  CeFusedArgs arg = a;
  void* args[] = {&arg};
  KernelTimer t(label ? K_CE_FUSED : K_CE_GUARD, s);
  const void* fn = fns[label ? 1 : 0][a.ksplit > 1 ? 1 : 0];
  return hipLaunchCooperativeKernel(fn, dim3(8 * kCeTeam), dim3(CfgBig::NT), args, (unsigned)kFusedLds, s);
}

hipError_t launch_ce_fused_status(const int* sync, int* gate, hipStream_t s) {
  hipLaunchKernelGGL(ce_fused_status_kernel, dim3(1), dim3(64), 0, s, sync, gate);
  return hipGetLastError();
}

hipError_t launch_ce_fused_nan(const int* sync, float* loss, int E, float* lse, int N, void* grad, int64_t nd,
                               hipStream_t s) {
  KernelTimer t(K_CE_GUARD, s);
  hipLaunchKernelGGL(ce_fused_nan_kernel, dim3(256), dim3(256), 0, s, sync, loss, E, lse, N,
                     static_cast<bf16_t*>(grad), nd);
  return hipGetLastError();
}

}  // namespace attt
