// The bf16 MFMA GEMM core shared by the LM-head kernels: tile order, tile configurations,
// buffer-descriptor loads and the two mainloops (plain double-buffered for 4 waves, ping-pong
// for 8 waves), accumulating acc += A[0:BM, 0:K] B[0:BN, 0:K]^T with both operands contiguous
// along K. MFMA v_mfma_f32_32x32x16_bf16, and the ping-pong also on v_mfma_f32_16x16x32_bf16.
#pragma once

#include "common.hpp"

namespace attt {

// ------------------------------------------------------------------------------------------
// Shared helpers
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int xcd = bid & 7, j = bid >> 3;
  const int q = total >> 3, r = total & 7;
  return xcd * q + min(xcd, r) + j;
}

// Tile of workgroup `bid`: each XCD takes a contiguous range of the tile order, and that
// order walks groups of 8 row tiles column by column, so the ~32 workgroups resident on one
// XCD cover about 8 row panels x 4 column panels and share them in that XCD's L2.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int t = xcd_remap(bid, tiles_m * tiles_n);
  constexpr int GM = 8;
  const int per_group = GM * tiles_n;
  const int g = t / per_group;
  const int first = g * GM;
  const int gm = min(GM, tiles_m - first);
  const int local = t - g * per_group;
  tm = first + local % gm;
  tn = local / gm;
}

// Workgroup tile BM x BN computed by WGM x WGN waves; each wave owns a (BM/WGM) x (BN/WGN)
// block of 32x32 MFMA tiles. K advances 64 per stage, two stages in LDS.
template <int BM_, int BN_, int WGM_, int WGN_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN;
  static constexpr int BK = 64;
  static constexpr int WTM = BM / WGM, WTN = BN / WGN;
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int RPL = NT / 8;  // rows one load round covers (8 x 16-byte chunks per row)
  static constexpr int AL = BM / RPL, BL = BN / RPL;
  static constexpr int SA = BM * BK, SB = BN * BK;
  static constexpr size_t LDS_STAGES = (size_t)2 * (SA + SB) * sizeof(bf16_t);  // two stages
  // + the ping-pong mainloops' group counter (256 bytes, so what a kernel puts after it stays aligned)
  static constexpr size_t LDS = LDS_STAGES + 256;
};
using CfgBig = Cfg<256, 256, 2, 4>;    // 8 waves, 128x64 per wave
using CfgSmall = Cfg<128, 128, 2, 2>;  // 4 waves, 64x64 per wave

// Buffer loads return zero for offsets past the descriptor's range: masked lanes use kOOB
// instead of branching. Valid offsets stay far below kRsrcBytes (a tile spans < 256 rows).
constexpr uint32_t kOOB = 0x7FFFFFF0u;
constexpr int kRsrcBytes = 0x40000000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p) { return buffer_rsrc(p, kRsrcBytes); }
__device__ __forceinline__ u32x4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// acc += A[0:BM, 0:K] * B[0:BN, 0:K]^T, A and B K-contiguous bf16. Rows at or past mval
// (nval) and K-chunks at or past K read as zero. K % 8 == 0.
template <class C>
__device__ __forceinline__ void mfma_mainloop_db(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                              const bf16_t* __restrict__ B, int64_t ldb, int nval,
                                              int K, bf16_t* lds, f32x16 (&acc)[C::TM][C::TN]) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
  const int wm = wave / C::WGN, wn = wave % C::WGN;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // Global -> LDS without registers: buffer_load_dwordx4 ... lds writes lane i's 16 bytes at
  // LDS base + 16 i, so one instruction fills a 1 KiB block of 8 rows x 128 bytes. Lane i of a
  // block takes row 8*block + i/8 and physical chunk i%8, and fetches the logical chunk that
  // the swizzle stores there (physical ^ (row/2)%8). The stage's blocks are dealt round-robin
  // to the waves.
  const __amdgpu_buffer_rsrc_t rA = make_rsrc(A), rB = make_rsrc(B);
  constexpr int NW = C::NT / 64;
  constexpr int ABLK = C::BM / 8, BBLK = C::BN / 8;
  constexpr int BPW = (ABLK + BBLK) / NW;  // blocks per wave per stage
  static_assert((ABLK + BBLK) % NW == 0 && ABLK % NW == 0, "stage blocks must split evenly");
  uint32_t goff[BPW];
  int gch[BPW];
#pragma unroll
  for (int j = 0; j < BPW; ++j) {
    const int blk = wave + j * NW;
    const bool isA = blk < ABLK;
    const int row = (isA ? blk : blk - ABLK) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    gch[j] = c;
    const int val = isA ? mval : nval;
    const int64_t ld = isA ? lda : ldb;
    goff[j] = row < val ? (uint32_t)((int64_t)row * ld * 2) + c * 16 : kOOB;
  }
  auto dma = [&](int st, int k0) {
    bf16_t* base = lds + st * (C::SA + C::SB);
    const uint32_t kb = (uint32_t)k0 * 2;
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
      const int blk = wave + j * NW;
      const bool isA = blk < ABLK;
      const bool kin = k0 + gch[j] * 8 < K;
      const uint32_t off = (kin && goff[j] != kOOB) ? goff[j] + kb : kOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isA ? rA : rB,
                                               (__attribute__((address_space(3))) void*)(base + blk * 512),
                                               16, off, 0, 0, 0);
    }
  };

  const int nk = (K + 63) / 64;
  dma(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  const int l32 = lane & 31, hi = lane >> 5;
  const int swz = (l32 >> 1) & 7;
  const int arow = (wm * C::WTM + l32) * 64, brow = (wn * C::WTN + l32) * 64;
  // operand fragments of sub-step kk live in fa/fb[kk & 1]; the reads for kk+1 are issued
  // before the MFMAs of kk so their LDS latency hides behind those MFMAs
  bf16x8 fa[2][C::TM], fb[2][C::TN];
  auto fragload = [&](const bf16_t* As, const bf16_t* Bs, int kk, int slot) {
    const int sw = ((kk * 2 + hi) ^ swz) << 3;
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
      fa[slot][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(As + arow + i * 32 * 64 + sw));
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
      fb[slot][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(Bs + brow + j * 32 * 64 + sw));
  };
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) dma((kt + 1) & 1, (kt + 1) * 64);
    const bf16_t* As = lds + (kt & 1) * (C::SA + C::SB);
    const bf16_t* Bs = As + C::SA;
    fragload(As, Bs, 0, 0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (kk + 1 < 4) fragload(As, Bs, kk + 1, (kk + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk & 1][i], fb[kk & 1][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of the next stage have landed in LDS
    __syncthreads();
  }
}

// 8-wave ping-pong schedule. Waves 0-3 and 4-7 form two groups with one wave of each on every
// SIMD. Phases are separated by workgroup barriers and group 1 runs one phase behind group 0, so
// in every phase one wave per SIMD reads a whole K-step of operand fragments from LDS (memory
// phase) while the other runs its 32 MFMAs (compute phase).
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// The group counter of the ping-pong mainloops: an int in LDS after the two stage buffers.
// group1_reset() zeroes it before a mainloop's first barrier (thread 0; the caller's wait for
// its LDS operations follows). Every wave of group 1 calls group1_arrive() once its fragment
// reads of stage k have completed (lgkmcnt(0)), and group1_wait(k) before it refills blocks the
// other waves of its group read: it returns once all four have arrived for stage k. All four
// run the same loop iterations, so the wait always ends. Both use inline LDS instructions: the
// compiler would otherwise wait for the wave's outstanding LDS-DMA loads (vmcnt) before them,
// since it cannot tell that the counter is not among their destinations.
template <class C>
__device__ __forceinline__ uint32_t group1_counter(bf16_t* lds) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)(reinterpret_cast<uint8_t*>(lds) +
                                                                        C::LDS_STAGES);
}
__device__ __forceinline__ void group1_reset(uint32_t ctr, int tid) {
  if (tid == 0) asm volatile("ds_write_b32 %0, %1" ::"v"(ctr), "v"(0) : "memory");
}
__device__ __forceinline__ void group1_arrive(uint32_t ctr, int lane) {
  if (lane == 0) asm volatile("ds_add_u32 %0, %1" ::"v"(ctr), "v"(1) : "memory");
}
__device__ __forceinline__ void group1_wait(uint32_t ctr, int k) {
  const int target = 4 * (k + 1);
  int v;
  do {
    asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(ctr) : "memory");
  } while (__builtin_amdgcn_readfirstlane(v) < target);
}

// Tile loads are issued only in memory phases: a wave stalls at a load instruction until the
// load path accepts it (about 1 KiB per 25 cycles per CU here), and a stall in a compute phase
// idles the SIMD's matrix core. A stage is 64 instructions of 1 KiB, 16 per wave of a group
// (j in [0, 16), see PpLoader); both groups share them:
//  * group 0 issues blocks [kSafe, kG1) of stage k+1 at the start of its memory phase of stage
//    k (slot (k+1)&1 was last read by group 1 in the phase before) and waits for them at the
//    end of its compute phase of stage k;
//  * group 1 issues the rest of stage k+2 into slot k&1 at the end of its memory phase of
//    stage k, after its own fragment reads of stage k have completed (group 0 finished reading
//    that slot before the barrier that opened the phase), and waits for them one memory phase
//    later: first blocks [0, kSafe), the A rows of group 0's half that no wave of group 1
//    reads, then, once all four waves of group 1 have read stage k (group1_wait), blocks
//    [kG1, 16). The four waves of group 1 read the same A rows and, pairwise with group 0, the
//    same B rows, so a wave that refilled those after its own reads only could overwrite them
//    before a slower wave of its group had read them (its fragments then came from stage k+2).
//    Issuing the safe blocks first keeps the wait behind load issue that is needed anyway.
// Group 1's share thus has three phases to land instead of one, and neither group's memory
// phase carries a whole stage of load issue.
// `tid` is the thread's index in the workgroup (a caller inside a loop may pass it through an
// empty asm so that the per-lane offsets derived from it are not hoisted out of that loop).
//
// The stage loads of the ping-pong mainloop: a stage's 64 blocks of 8 rows x 128 bytes are block
// (wave & 3) + 4 j for j in [0, 16). Blocks j < 8 are A rows, the rest B rows; both groups use the
// same numbering. Offsets are formed per load: the block's first row is wave-uniform, and the
// swizzled chunk of a lane depends only on the lane and on the parity of the block.
// The stage buffers start at the kernel's LDS address 0 (the kernels declare no static LDS) and
// are followed by the group counter at byte LDS_STAGES.
template <class C>
struct PpLoader {
  static constexpr int LW = 4;                        // waves per group
  static constexpr int ABLK = C::BM / 8, BBLK = C::BN / 8;
  static constexpr int BPW = (ABLK + BBLK) / LW;      // blocks per wave of a group per stage
  static constexpr int kSafe = C::WTM / 8 / LW;       // j < kSafe: A rows of group 0's half only
  static constexpr int kG1 = kSafe + 6;               // group 0's share: j in [kSafe, kG1)
  static_assert(ABLK % LW == 0 && BBLK % LW == 0 && kG1 < BPW, "stage blocks must split evenly");
  static_assert(C::WGM == 2 && C::WGN == LW, "waves 0-3 cover A rows [0, WTM), waves 4-7 the rest");
  __amdgpu_buffer_rsrc_t rA, rB;
  int64_t lda, ldb;
  int mval, nval, K, wave, lr, c_even, c_odd;
  uint32_t la, lb;
  __device__ __forceinline__ PpLoader(const bf16_t* A, int64_t lda_, int mval_, const bf16_t* B, int64_t ldb_,
                                      int nval_, int K_, int tid)
      : rA(make_rsrc(A)), rB(make_rsrc(B)), lda(lda_), ldb(ldb_), mval(mval_), nval(nval_), K(K_) {
    const int lane = tid & 63;
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    lr = lane >> 3;
    c_even = (lane & 7) ^ ((lr >> 1) & 7);
    c_odd = (lane & 7) ^ (((8 + lr) >> 1) & 7);
    la = (uint32_t)(lr * lda * 2);
    lb = (uint32_t)(lr * ldb * 2);
  }
  // blocks j in [j0, j1) of this wave for the stage at K offset k0, into LDS stage buffer st
  __device__ __forceinline__ void issue(bf16_t* lds, int st, int k0, int j0, int j1) const {
    bf16_t* base = lds + st * (C::SA + C::SB);
#pragma unroll
    for (int j = j0; j < j1; ++j) {
      const int blk = (wave & 3) + j * LW;
      const bool isA = blk < ABLK;
      const int rb = (isA ? blk : blk - ABLK) * 8;
      const int c = (rb & 8) ? c_odd : c_even;
      const bool ok = rb + lr < (isA ? mval : nval) && k0 + c * 8 < K;
      const uint32_t off = (uint32_t)((int64_t)rb * (isA ? lda : ldb) * 2) + (isA ? la : lb) +
                           (uint32_t)(k0 + c * 8) * 2;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isA ? rA : rB,
                                               (__attribute__((address_space(3))) void*)(base + blk * 512),
                                               16, ok ? off : kOOB, 0, 0, 0);
    }
  }
  // group 1's share of a stage: blocks [0, kSafe) and [kG1, BPW)
  __device__ __forceinline__ void issue_group1(bf16_t* lds, int st, int k0) const {
    issue(lds, st, k0, 0, kSafe);
    issue(lds, st, k0, kG1, BPW);
  }
  // the loads that precede the loop: group 0 all of stage 0, group 1 its share of stage 1
  __device__ __forceinline__ void prologue(bf16_t* lds, bool wait_between) const {
    const int grp = wave >> 2;
    if (grp == 0) issue(lds, 0, 0, 0, BPW);
    if (wait_between) __builtin_amdgcn_s_waitcnt(0);
    if (grp == 1 && K > 64) issue_group1(lds, 1, 64);
  }
};

// Issues the ping-pong mainloop's prologue loads for a later call with `issued` set: a caller
// can start the next tile's first stages before it spends time on this tile's epilogue. The
// LDS stage buffers must be free (the previous mainloop has returned) and must stay untouched
// until that call.
template <class C>
__device__ __forceinline__ void mfma_pp_prologue(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                                 const bf16_t* __restrict__ B, int64_t ldb, int nval, int K,
                                                 bf16_t* lds, int tid) {
  PpLoader<C>(A, lda, mval, B, ldb, nval, K, tid).prologue(lds, false);
}

template <class C>
__device__ __forceinline__ void mfma_mainloop_pp(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                                 const bf16_t* __restrict__ B, int64_t ldb, int nval,
                                                 int K, bf16_t* lds, f32x16 (&acc)[C::TM][C::TN],
                                                 int tid = (int)threadIdx.x, bool issued = false) {
  static_assert(C::NT == 512 && C::WGM == 2 && C::WGN == 4, "ping-pong needs 8 waves in 2 groups of 4");
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int grp = wave >> 2;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const PpLoader<C> ld(A, lda, mval, B, ldb, nval, K, tid);
  constexpr int BPW = PpLoader<C>::BPW, kSafe = PpLoader<C>::kSafe, kG1 = PpLoader<C>::kG1;

  const int l32 = lane & 31, hi = lane >> 5;
  const int swz = (l32 >> 1) & 7;
  const int arow = (wm * C::WTM + l32) * 64, brow = (wn * C::WTN + l32) * 64;
  bf16x8 fa[4][C::TM], fb[4][C::TN];
  auto mem = [&](int k) {
    const bf16_t* As = lds + (k & 1) * (C::SA + C::SB);
    const bf16_t* Bs = As + C::SA;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int sw = ((kk * 2 + hi) ^ swz) << 3;
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
        fa[kk][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(As + arow + i * 32 * 64 + sw));
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
        fb[kk][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(Bs + brow + j * 32 * 64 + sw));
    }
  };
  auto compute = [&]() {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk][i], fb[kk][j], acc[i][j], 0, 0, 0);
  };
  // MFMAs are pure register operations and could be moved across the barriers; tying the
  // accumulators to empty asm statements keeps each compute phase between its two barriers.
  auto pin = [&]() {
    static_assert(C::TM == 4 && C::TN == 2, "pin lists the 8 accumulators of a 128x64 wave tile");
    asm volatile("" : "+v"(acc[0][0]), "+v"(acc[0][1]), "+v"(acc[1][0]), "+v"(acc[1][1]),
                 "+v"(acc[2][0]), "+v"(acc[2][1]), "+v"(acc[3][0]), "+v"(acc[3][1]));
  };
  // Group 0, iteration k:  loads [kSafe, kG1) of stage k+1; fragments(k); wait for own reads |
  //                        MFMA(k); wait for own loads |
  // group 1, one phase later: fragments(k); wait for own reads and loads; loads [0, kSafe) of
  //                        stage k+2; wait for the group's reads; loads [kG1, 16) | MFMA(k) |
  // Group 1 takes one extra barrier before its loop, group 0 one after it, so every wave
  // executes 2 nk + 2 barriers. Group 1's share of stage 1 is issued before the loop (with
  // `issued`, the caller has issued both prologue loads already, see mfma_pp_prologue).
  const int nk = (K + 63) / 64;
  const uint32_t ctr = group1_counter<C>(lds);
  group1_reset(ctr, tid);
  if (!issued) ld.prologue(lds, true);
  else if (grp == 0) __builtin_amdgcn_s_waitcnt(0);  // stage 0 has landed (group 1 waits in its loop)
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the counter reset has landed
  wg_barrier();
  if (grp == 0) {
    for (int k = 0; k < nk; ++k) {
      if (k + 1 < nk) ld.issue(lds, (k + 1) & 1, (k + 1) * 64, kSafe, kG1);
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
      if (k + 2 < nk) {
        group1_arrive(ctr, lane);
        ld.issue(lds, k & 1, (k + 2) * 64, 0, kSafe);
        group1_wait(ctr, k);
        ld.issue(lds, k & 1, (k + 2) * 64, kG1, BPW);
      }
      wg_barrier();
      pin();
      compute();
      pin();
      wg_barrier();
    }
  }
}

// ------------------------------------------------------------------------------------------
// The same 8-wave ping-pong on v_mfma_f32_16x16x32_bf16. A wave's 128 x 64 block is 8 x 4 tiles
// of 16 x 16; register r of lane l of a tile holds row 4 (l / 16) + r, column l % 16 (Mma16).
// Per FLOP this moves fewer accumulator bytes through the register file than the 32x32x16
// form, and the chip holds a higher clock for the same work.
// ------------------------------------------------------------------------------------------
struct Mma16 {
  static constexpr int TM = 8, TN = 4;  // 16 x 16 tiles of a 128 x 64 wave block
  __device__ static __forceinline__ int row(int r, int lane) { return ((lane >> 4) << 2) + r; }
  __device__ static __forceinline__ int col(int lane) { return lane & 15; }
};
using Acc16 = f32x4[Mma16::TM][Mma16::TN];

// Fragments of one K-step (64) from an LDS stage: two K-halves of 32; lane l reads row
// (l % 16) of each 16-row tile at K chunk 4 kk + l / 16 (8 bf16), through the stage's swizzle.
template <class C>
__device__ __forceinline__ void mma16_frags(const bf16_t* As, const bf16_t* Bs, int lane, int wm, int wn,
                                            bf16x8 (&fa)[2][Mma16::TM], bf16x8 (&fb)[2][Mma16::TN]) {
  static_assert(C::WTM == 16 * Mma16::TM && C::WTN == 16 * Mma16::TN, "128 x 64 wave blocks");
  const int l16 = lane & 15, q4 = lane >> 4, swz = (l16 >> 1) & 7;
  const int arow = (wm * C::WTM + l16) * 64, brow = (wn * C::WTN + l16) * 64;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int sw = ((kk * 4 + q4) ^ swz) << 3;
#pragma unroll
    for (int i = 0; i < Mma16::TM; ++i)
      fa[kk][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(As + arow + i * 16 * 64 + sw));
#pragma unroll
    for (int j = 0; j < Mma16::TN; ++j)
      fb[kk][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(Bs + brow + j * 16 * 64 + sw));
  }
}

__device__ __forceinline__ void mma16_step(const bf16x8 (&fa)[2][Mma16::TM], const bf16x8 (&fb)[2][Mma16::TN],
                                           Acc16& acc) {
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int i = 0; i < Mma16::TM; ++i)
#pragma unroll
      for (int j = 0; j < Mma16::TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[kk][i], fb[kk][j], acc[i][j], 0, 0, 0);
}

// Ties the accumulators to empty asm statements so that the MFMAs between two pins stay between
// the barriers around them (MFMAs touch no memory; the compiler could move them across).
__device__ __forceinline__ void mma16_pin(Acc16& acc) {
  static_assert(Mma16::TM == 8 && Mma16::TN == 4, "pins list 32 accumulators");
  asm volatile("" : "+v"(acc[0][0]), "+v"(acc[0][1]), "+v"(acc[0][2]), "+v"(acc[0][3]), "+v"(acc[1][0]),
               "+v"(acc[1][1]), "+v"(acc[1][2]), "+v"(acc[1][3]), "+v"(acc[2][0]), "+v"(acc[2][1]),
               "+v"(acc[2][2]), "+v"(acc[2][3]), "+v"(acc[3][0]), "+v"(acc[3][1]), "+v"(acc[3][2]),
               "+v"(acc[3][3]));
  asm volatile("" : "+v"(acc[4][0]), "+v"(acc[4][1]), "+v"(acc[4][2]), "+v"(acc[4][3]), "+v"(acc[5][0]),
               "+v"(acc[5][1]), "+v"(acc[5][2]), "+v"(acc[5][3]), "+v"(acc[6][0]), "+v"(acc[6][1]),
               "+v"(acc[6][2]), "+v"(acc[6][3]), "+v"(acc[7][0]), "+v"(acc[7][1]), "+v"(acc[7][2]),
               "+v"(acc[7][3]));
}

// mfma_mainloop_pp with 16x16x32 MFMAs: the same loads, barriers and phases.
template <class C>
__device__ __forceinline__ void mfma_mainloop_pp16(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                                   const bf16_t* __restrict__ B, int64_t ldb, int nval, int K,
                                                   bf16_t* lds, Acc16& acc, int tid = (int)threadIdx.x,
                                                   bool issued = false) {
  static_assert(C::NT == 512 && C::WGM == 2 && C::WGN == 4, "ping-pong needs 8 waves in 2 groups of 4");
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int grp = wave >> 2;
#pragma unroll
  for (int i = 0; i < Mma16::TM; ++i)
#pragma unroll
    for (int j = 0; j < Mma16::TN; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  const PpLoader<C> ld(A, lda, mval, B, ldb, nval, K, tid);
  constexpr int BPW = PpLoader<C>::BPW, kSafe = PpLoader<C>::kSafe, kG1 = PpLoader<C>::kG1;
  bf16x8 fa[2][Mma16::TM], fb[2][Mma16::TN];
  auto mem = [&](int k) {
    const bf16_t* As = lds + (k & 1) * (C::SA + C::SB);
    mma16_frags<C>(As, As + C::SA, lane, wm, wn, fa, fb);
  };
  const int nk = (K + 63) / 64;
  const uint32_t ctr = group1_counter<C>(lds);
  group1_reset(ctr, tid);
  if (!issued) ld.prologue(lds, true);
  else if (grp == 0) __builtin_amdgcn_s_waitcnt(0);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the counter reset has landed
  wg_barrier();
  if (grp == 0) {
    for (int k = 0; k < nk; ++k) {
      if (k + 1 < nk) ld.issue(lds, (k + 1) & 1, (k + 1) * 64, kSafe, kG1);
      mem(k);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();
      mma16_pin(acc);
      mma16_step(fa, fb, acc);
      mma16_pin(acc);
      __builtin_amdgcn_s_waitcnt(0);
      wg_barrier();
    }
    wg_barrier();
  } else {
    wg_barrier();
    for (int k = 0; k < nk; ++k) {
      mem(k);
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      if (k + 2 < nk) {
        group1_arrive(ctr, lane);
        ld.issue(lds, k & 1, (k + 2) * 64, 0, kSafe);
        group1_wait(ctr, k);
        ld.issue(lds, k & 1, (k + 2) * 64, kG1, BPW);
      }
      wg_barrier();
      mma16_pin(acc);
      mma16_step(fa, fb, acc);
      mma16_pin(acc);
      wg_barrier();
    }
  }
}

template <class C>
__device__ __forceinline__ void mfma_mainloop(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                              const bf16_t* __restrict__ B, int64_t ldb, int nval,
                                              int K, bf16_t* lds, f32x16 (&acc)[C::TM][C::TN]) {
  if constexpr (C::NT == 512)
    mfma_mainloop_pp<C>(A, lda, mval, B, ldb, nval, K, lds, acc);
  else
    mfma_mainloop_db<C>(A, lda, mval, B, ldb, nval, K, lds, acc);
}

// Output layout of a 32x32 MFMA accumulator: register r of lane l holds
// row 8*(r/4) + 4*(l/32) + r%4, column l%32.
__device__ __forceinline__ int mfma_row(int r, int lane) { return ((r >> 2) << 3) + ((lane >> 5) << 2) + (r & 3); }

}  // namespace attt
