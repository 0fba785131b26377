// Token-weighted cross-entropy through a frozen LM head (Sec. 3.3, Eq. 10), forward and
// backward with respect to the hidden states, on gfx950.
//
// Forward only (logits never leave the chip): one GEMM z = h W^T over (vocab tile, row tile)
// whose epilogue reduces every row of the tile to (max, sum exp(z - max)). A row kernel merges
// the partials into lse and w * CE; an episode kernel sums those in a fixed order into
// loss_e = (1/L_e) sum w_t CE_t.
//
// Forward + backward (bf16): two GEMMs over the vocabulary, the algorithmic 4 N V d flops.
// Every row takes its own label logit r_t = z_{t,y_t} as the exponent reference, so the first
// GEMM can form e_tv = exp(z_tv - r_t) without knowing lse:
//     sigma_t = sum_{v != y_t} e_tv,   lse_t = r_t + log1p(sigma_t),   CE_t = log1p(sigma_t)
//     dL/dh_t = (w_t / L_e) (U_t - sigma_t W_{y_t}) / (1 + sigma_t),  U_t = sum_{v != y_t} e_tv W_v
// which is (w_t / L_e)(softmax(z_t) - onehot(y_t)) W rewritten; the label term is kept out of
// the sums, so nothing cancels when p_y is close to 1. Per vocab chunk, the first GEMM
// (ce_logit_exp) stores e (bf16) into a bounded staging buffer and the per-row sums of its
// tile; the second (ce_bwd_dh) accumulates U += e_chunk W_chunk in float32. After the last
// chunk's first GEMM a row kernel forms sigma, lse and CE, and the last dh epilogue applies
// the row scale and the label term. r_t is one of the row's logits, so sigma never
// underflows; a logit more than 64 above r_t (a label with probability below e^-64)
// could overflow e, and sets a flag on which the exact three-GEMM path (forward lse, then
// dZ = (w/L)(exp(z - lse) - onehot) and dH = dZ W) reruns in full, overwriting the outputs.
// Its kernels read the flag first and return at once when it is clear.
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16. A 256x256 tile runs on 8 waves (2x4, 128x64
// each, two waves per SIMD); small problems use 128x128 on 4 waves. K advances 64 per stage,
// double-buffered in LDS, with an XOR swizzle of the 16-byte chunks (chunk ^ (row/2)%8): the
// LDS serves 16 lanes of a 16-byte read per clock over 64 banks, and the 16 consecutive rows
// those lanes read fall in distinct banks. Global reads are buffer loads whose masked lanes
// point past the descriptor's range (the hardware returns zero, no branches). Tile order is
// XCD-aware: workgroup i runs on XCD i%8, each XCD takes a contiguous range of the order, and
// the order walks groups of 8 row tiles column by column, so the workgroups resident on one
// XCD share a few hidden and LM-head panels in its L2.
// f32 path: plain VALU tiles (64x64, 4x4 per thread) running the three-GEMM algorithm; it
// serves the float32 configuration.
#include "common.hpp"
#include "internal.hpp"

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
  static constexpr size_t LDS = (size_t)2 * (SA + SB) * sizeof(bf16_t);  // two stages
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

// Tile loads are issued only in memory phases: a wave stalls at a load instruction until the
// load path accepts it (about 1 KiB per 25 cycles per CU here), and a stall in a compute phase
// idles the SIMD's matrix core. A stage is 64 instructions of 1 KiB; both groups share them:
//  * group 0 issues blocks [0, kG0) of stage k+1 at the start of its memory phase of stage k
//    (slot (k+1)&1 was last read by group 1 in the phase before) and waits for them at the end
//    of its compute phase of stage k;
//  * group 1 issues blocks [kG0, 16) of stage k+2 at the end of its memory phase of stage k,
//    after its own fragment reads of slot k&1 have completed (group 0 finished reading that
//    slot before the barrier that opened the phase), and waits for them one memory phase later.
// Group 1's share thus has three phases to land instead of one, and neither group's memory
// phase carries a whole stage of load issue.
template <class C>
__device__ __forceinline__ void mfma_mainloop_pp(const bf16_t* __restrict__ A, int64_t lda, int mval,
                                                 const bf16_t* __restrict__ B, int64_t ldb, int nval,
                                                 int K, bf16_t* lds, f32x16 (&acc)[C::TM][C::TN]) {
  static_assert(C::NT == 512 && C::WGM == 2 && C::WGN == 4, "ping-pong needs 8 waves in 2 groups of 4");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int grp = wave >> 2;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // A stage's 64 blocks of 8 rows x 128 bytes: block (wave & 3) + 4 j for j in [0, 16). Blocks
  // j < 8 are A rows, the rest B rows; both groups use the same numbering.
  const __amdgpu_buffer_rsrc_t rA = make_rsrc(A), rB = make_rsrc(B);
  constexpr int LW = 4;                               // waves per group
  constexpr int ABLK = C::BM / 8, BBLK = C::BN / 8;
  constexpr int BPW = (ABLK + BBLK) / LW;             // blocks per wave of a group per stage
  constexpr int kG0 = 6;                              // group 0's share per wave
  static_assert(ABLK % LW == 0 && BBLK % LW == 0 && kG0 < BPW, "stage blocks must split evenly");
  // Offsets are formed per load: the block's first row is wave-uniform, and the swizzled chunk
  // of a lane depends only on the lane and on the parity of the block (rows 8b .. 8b+7).
  const int lr = lane >> 3;
  const int c_even = (lane & 7) ^ ((lr >> 1) & 7);
  const int c_odd = (lane & 7) ^ (((8 + lr) >> 1) & 7);
  const uint32_t la = (uint32_t)(lr * lda * 2), lb = (uint32_t)(lr * ldb * 2);
  auto dma = [&](int st, int k0, int j0, int j1) {
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
  };

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
  // Group 0, iteration k:  loads [0, kG0) of stage k+1; fragments(k); wait for own reads |
  //                        MFMA(k); wait for own loads |
  // group 1, one phase later: fragments(k); wait for own reads and loads; loads [kG0, 16) of
  //                        stage k+2 | MFMA(k) |
  // Group 1 takes one extra barrier before its loop, group 0 one after it, so every wave
  // executes 2 nk + 2 barriers. Group 1's share of stage 1 is issued before the loop.
  const int nk = (K + 63) / 64;
  if (grp == 0) dma(0, 0, 0, BPW);
  __builtin_amdgcn_s_waitcnt(0);
  if (grp == 1 && nk > 1) dma(1, 64, kG0, BPW);
  wg_barrier();
  if (grp == 0) {
    for (int k = 0; k < nk; ++k) {
      if (k + 1 < nk) dma((k + 1) & 1, (k + 1) * 64, 0, kG0);
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
      if (k + 2 < nk) dma(k & 1, (k + 2) * 64, kG0, BPW);
      wg_barrier();
      pin();
      compute();
      pin();
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

// ------------------------------------------------------------------------------------------
// bf16 forward. The GEMM runs transposed, z^T = W h^T, so a workgroup tile is 256 vocab rows x
// 256 token columns and every lane holds, for one token, 64 of the tile's vocab logits in its
// registers: the per-token (max, sum exp) needs one cross-lane step (lanes l and l+32) and a
// two-wave merge in LDS, instead of a 32-lane shuffle tree per row.
// ------------------------------------------------------------------------------------------
template <class C>
__device__ __forceinline__ void ce_fwd_bf16_body(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, int N, int d, int V, int tiles_v,
    int tiles_t, float2* __restrict__ partials, int n_vb) {
  extern __shared__ __align__(16) uint8_t smem[];
  int tv, tt;
  tile_of(blockIdx.x, tiles_v, tiles_t, tv, tt);
  const int v0 = tv * C::BM, t0 = tt * C::BN;
  f32x16 acc[C::TM][C::TN];
  mfma_mainloop<C>(W + (int64_t)v0 * d, d, V - v0, h + (int64_t)t0 * d, d, N - t0, d,
                   reinterpret_cast<bf16_t*>(smem), acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  float* red_m = reinterpret_cast<float*>(smem);  // [WGM][BN]
  float* red_s = red_m + C::WGM * C::BN;
  const int vbase = v0 + wm * C::WTM;
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (vbase + i * 32 + mfma_row(r, lane) < V) mx = fmaxf(mx, acc[i][j][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float s = 0.0f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (vbase + i * 32 + mfma_row(r, lane) < V) s += __expf(acc[i][j][r] - mx);
    }
    s += __shfl_xor(s, 32, 64);
    if (lane < 32) {
      const int tl = wn * C::WTN + j * 32 + lane;
      red_m[wm * C::BN + tl] = mx;
      red_s[wm * C::BN + tl] = s;
    }
  }
  __syncthreads();
  for (int tl = threadIdx.x; tl < C::BN; tl += C::NT) {
    const int t = t0 + tl;
    if (t >= N) continue;
    float m = red_m[tl], s = red_s[tl];
#pragma unroll
    for (int w = 1; w < C::WGM; ++w) lse_merge(m, s, red_m[w * C::BN + tl], red_s[w * C::BN + tl]);
    partials[(int64_t)t * n_vb + tv] = make_float2(m, s);
  }
}

template <class C>
__global__ __launch_bounds__(C::NT) void ce_fwd_bf16_kernel(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, int N, int d, int V, int tiles_v,
    int tiles_t, float2* __restrict__ partials, int n_vb) {
  ce_fwd_bf16_body<C>(h, W, N, d, V, tiles_v, tiles_t, partials, n_vb);
}

// The same kernel launched by the overflow guard: returns at once unless *gate != 0.
template <class C>
__global__ __launch_bounds__(C::NT) void ce_guard_fwd_bf16_kernel(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, int N, int d, int V, int tiles_v,
    int tiles_t, float2* __restrict__ partials, int n_vb, const int* __restrict__ gate) {
  if (*gate == 0) return;
  ce_fwd_bf16_body<C>(h, W, N, d, V, tiles_v, tiles_t, partials, n_vb);
}

// Label logit z_{t, y_t} = h_t . W_{y_t} (float32 accumulation), one wave per row.
__global__ __launch_bounds__(256) void ce_label_logit_bf16_kernel(const bf16_t* __restrict__ h,
                                                                  const bf16_t* __restrict__ W,
                                                                  const int32_t* __restrict__ labels,
                                                                  int N, int d, int V,
                                                                  float* __restrict__ label_logit,
                                                                  int* __restrict__ flag) {
  const int lane = threadIdx.x & 63;
  if (flag && blockIdx.x == 0 && threadIdx.x == 0) *flag = 0;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  const int y = labels[row];
  if (y < 0 || y >= V) {  // outside the contract: make the loss NaN instead of reading out of bounds
    if (lane == 0) label_logit[row] = __int_as_float(0x7FC00000);
    return;
  }
  const bf16_t* hr = h + (int64_t)row * d;
  const bf16_t* wr = W + (int64_t)y * d;
  float s = 0.0f;
  for (int k = lane * 8; k < d; k += 64 * 8) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(hr + k);
    const u32x4 b = *reinterpret_cast<const u32x4*>(wr + k);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      s = fmaf(bf16_bits_to_f32(a[e] & 0xFFFFu), bf16_bits_to_f32(b[e] & 0xFFFFu), s);
      s = fmaf(bf16_bits_to_f32(a[e] >> 16), bf16_bits_to_f32(b[e] >> 16), s);
    }
  }
  s = group_sum<64>(s);
  if (lane == 0) label_logit[row] = s;
}

// bf16 backward part 1: dZ for rows [r0, r0+R) x vocab [c0, c0 + tiles_n*BN) into staging.
template <class C>
__device__ __forceinline__ void ce_dz_bf16_body(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, const int32_t* __restrict__ labels,
    const float* __restrict__ lse, const float* __restrict__ coef, int r0, int R, int d, int c0,
    int cend, int V, int tiles_m, int tiles_n, bf16_t* __restrict__ dz, int ldz) {
  extern __shared__ __align__(16) uint8_t smem[];
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * C::BM, n0 = tn * C::BN;
  f32x16 acc[C::TM][C::TN];
  mfma_mainloop<C>(h + (int64_t)(r0 + m0) * d, d, R - m0, W + (int64_t)(c0 + n0) * d, d,
                   cend - (c0 + n0), d, reinterpret_cast<bf16_t*>(smem), acc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
#pragma unroll
  for (int i = 0; i < C::TM; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = m0 + wm * C::WTM + i * 32 + mfma_row(r, lane);
      if (rl >= R) continue;
      const int row = r0 + rl;
      const float l = lse[row], c = coef[row];
      const int y = labels[row];
#pragma unroll
      for (int j = 0; j < C::TN; ++j) {
        const int cl = n0 + wn * C::WTN + j * 32 + (lane & 31);
        const int col = c0 + cl;
        float g = 0.0f;
        if (col < V) g = c * (__expf(acc[i][j][r] - l) - (col == y ? 1.0f : 0.0f));
        dz[(int64_t)rl * ldz + cl] = (bf16_t)f32_to_bf16_bits(g);
      }
    }
  }
}

template <class C>
__global__ __launch_bounds__(C::NT) void ce_dz_bf16_kernel(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, const int32_t* __restrict__ labels,
    const float* __restrict__ lse, const float* __restrict__ coef, int r0, int R, int d, int c0,
    int cend, int V, int tiles_m, int tiles_n, bf16_t* __restrict__ dz, int ldz) {
  ce_dz_bf16_body<C>(h, W, labels, lse, coef, r0, R, d, c0, cend, V, tiles_m, tiles_n, dz, ldz);
}

// The same kernel launched by the overflow guard: returns at once unless *gate != 0.
template <class C>
__global__ __launch_bounds__(C::NT) void ce_guard_dz_bf16_kernel(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, const int32_t* __restrict__ labels,
    const float* __restrict__ lse, const float* __restrict__ coef, int r0, int R, int d, int c0,
    int cend, int V, int tiles_m, int tiles_n, bf16_t* __restrict__ dz, int ldz,
    const int* __restrict__ gate) {
  if (*gate == 0) return;
  ce_dz_bf16_body<C>(h, W, labels, lse, coef, r0, R, d, c0, cend, V, tiles_m, tiles_n, dz, ldz);
}

// bf16 backward part 2, transposed like the forward: acc[n, t] (+)= sum_k WT[n, c0 + k] S[t, k]
// over the staged chunk S (n a column of dH, t a row of the block), so every lane holds one
// row t and runs of four consecutive columns. The last chunk writes dH: acc itself (S = dZ),
// or, with row scales (S = e), dH_t = sa_t acc_t - sb_t W_{y_t} (sa = coef / (1 + sigma),
// sb = coef sigma / (1 + sigma)), as 32-byte stores.
template <class C>
__device__ __forceinline__ void ce_dh_bf16_body(
    const bf16_t* __restrict__ dz, int ldz, const bf16_t* __restrict__ WT, int Vp, int r0, int R,
    int d, int c0, int K, int tiles_m, int tiles_n, float* __restrict__ accbuf,
    bf16_t* __restrict__ grad, int first, int last, const float* __restrict__ sa,
    const float* __restrict__ sb, const int32_t* __restrict__ labels, const bf16_t* __restrict__ W,
    int V) {
  extern __shared__ __align__(16) uint8_t smem[];
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * C::BM, n0 = tn * C::BN;  // m0: first column of dH, n0: first row of the block
  f32x16 acc[C::TM][C::TN];
  mfma_mainloop<C>(WT + (int64_t)m0 * Vp + c0, Vp, d - m0, dz + (int64_t)n0 * ldz, ldz, R - n0, K,
                         reinterpret_cast<bf16_t*>(smem), acc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  // The float32 partial sums between chunks keep the accumulators' register layout: per tile,
  // per (MFMA tile i, j, quarter q of the 16 registers), the workgroup's threads hold 16
  // contiguous bytes each, so every read and write is a coalesced 16-byte access. Every launch
  // of one call uses the same tiling, so a tile reads back exactly what it wrote.
  // Buffer accesses: the per-slot offset is a scalar, the lane's offset the only vector operand.
  // The first chunk reads through an empty range (zeros), so the add needs no branch.
  float* tbase = accbuf + (size_t)(tm * tiles_n + tn) * (C::BM * C::BN);
  const __amdgpu_buffer_rsrc_t racc = buffer_rsrc(tbase, C::BM * C::BN * 4);
  const __amdgpu_buffer_rsrc_t rprev = buffer_rsrc(tbase, first ? 0 : C::BM * C::BN * 4);
  const uint32_t voff = threadIdx.x * 16u;
  auto soff = [](int i, int j, int q) { return (uint32_t)(((i * C::TN + j) * 4 + q) * C::NT * 16); };
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 p = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rprev, voff, soff(i, j, q), 0));
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += p[e];
      }
      __builtin_amdgcn_sched_barrier(0);  // one MFMA tile's partials in flight at a time: no spills
    }
  if (!last) {
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), racc, voff, soff(i, j, q), 0);
        }
    return;
  }
  const int hi = lane >> 5;
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    const int tl = n0 + wn * C::WTN + j * 32 + (lane & 31);  // row of the block
    const bool tok = tl < R;
    float a = 1.0f, b = 0.0f;
    const bf16_t* wy = nullptr;
    if (tok && sa) {
      const int row = r0 + tl;
      a = sa[row];
      b = sb[row];
      const int y = labels[row];
      if (y >= 0 && y < V) wy = W + (int64_t)y * d;
      else a = __int_as_float(0x7FC00000);  // outside the contract: NaN row, no read
    }
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      const int cb = m0 + wm * C::WTM + i * 32;  // column of the MFMA tile's first row
      // register r holds column cb + 8 (r/4) + 4 (lane/32) + r%4: four runs of four columns
      uint32_t pk[8];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = cb + 8 * g + 4 * hi;
        float wv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (wy && c + 4 <= d) {
          const uint2 u = *reinterpret_cast<const uint2*>(wy + c);
          wv[0] = bf16_bits_to_f32(u.x & 0xFFFFu);
          wv[1] = bf16_bits_to_f32(u.x >> 16);
          wv[2] = bf16_bits_to_f32(u.y & 0xFFFFu);
          wv[3] = bf16_bits_to_f32(u.y >> 16);
        }
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = a * acc[i][j][4 * g + e] - b * wv[e];
        pk[2 * g] = pack_bf16x2(v[0], v[1]);
        pk[2 * g + 1] = pack_bf16x2(v[2], v[3]);
      }
      // same half-wave exchange as the first GEMM: low lanes get columns 0-15, high 16-31
      uint32_t P[4] = {pk[0], pk[1], pk[2], pk[3]}, Q[4] = {pk[4], pk[5], pk[6], pk[7]};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const auto sw = __builtin_amdgcn_permlane32_swap(P[k], Q[k], false, false);
        P[k] = sw[0];
        Q[k] = sw[1];
      }
      const int c0w = cb + 16 * hi;  // d % 8 == 0: a run of 16 is whole, half, or absent
      if (tok && c0w + 8 <= d) {
        u32x4* dst = reinterpret_cast<u32x4*>(grad + (int64_t)(r0 + tl) * d + c0w);
        dst[0] = u32x4{P[0], P[1], Q[0], Q[1]};
        if (c0w + 16 <= d) dst[1] = u32x4{P[2], P[3], Q[2], Q[3]};
      }
    }
  }
}

template <class C>
__global__ __launch_bounds__(C::NT) void ce_dh_bf16_kernel(
    const bf16_t* __restrict__ dz, int ldz, const bf16_t* __restrict__ WT, int Vp, int r0, int R,
    int d, int c0, int K, int tiles_m, int tiles_n, float* __restrict__ accbuf,
    bf16_t* __restrict__ grad, int first, int last, const float* __restrict__ sa,
    const float* __restrict__ sb, const int32_t* __restrict__ labels, const bf16_t* __restrict__ W,
    int V) {
  ce_dh_bf16_body<C>(dz, ldz, WT, Vp, r0, R, d, c0, K, tiles_m, tiles_n, accbuf, grad, first, last,
                     sa, sb, labels, W, V);
}

// The same kernel launched by the overflow guard: returns at once unless *gate != 0.
template <class C>
__global__ __launch_bounds__(C::NT) void ce_guard_dh_bf16_kernel(
    const bf16_t* __restrict__ dz, int ldz, const bf16_t* __restrict__ WT, int Vp, int r0, int R,
    int d, int c0, int K, int tiles_m, int tiles_n, float* __restrict__ accbuf,
    bf16_t* __restrict__ grad, int first, int last, const float* __restrict__ sa,
    const float* __restrict__ sb, const int32_t* __restrict__ labels, const bf16_t* __restrict__ W,
    int V, const int* __restrict__ gate) {
  if (*gate == 0) return;
  ce_dh_bf16_body<C>(dz, ldz, WT, Vp, r0, R, d, c0, K, tiles_m, tiles_n, accbuf, grad, first, last,
                     sa, sb, labels, W, V);
}

// bf16 backward part 1, label-referenced: the chunk's logits transposed (vocab rows x token
// columns, as in the forward), then for token t (local row of the block), with r_t its label
// logit, e_tv = exp(z_tv - r_t) for v != y_t and v < V, zero otherwise. e goes in bf16 into
// staging [R, ldz] (vocab contiguous), each lane storing 32 bytes per MFMA tile after one
// half-wave exchange; the tile's per-token sum of e (float32) goes to sig_part[t][vocab tile].
// A lane whose sum of e exceeds e^64 sets *flag.

template <class C>
__global__ __launch_bounds__(C::NT) void ce_logit_exp_bf16_kernel(
    const bf16_t* __restrict__ h, const bf16_t* __restrict__ W, const int32_t* __restrict__ labels,
    const float* __restrict__ label_logit, int r0, int R, int d, int c0, int cend, int tiles_v,
    int tiles_t, float* __restrict__ sig_part, int n_vb, bf16_t* __restrict__ ez, int ldz,
    int* __restrict__ flag) {
  extern __shared__ __align__(16) uint8_t smem[];
  int tv, tt;
  tile_of(blockIdx.x, tiles_v, tiles_t, tv, tt);
  const int v0 = c0 + tv * C::BM, t0 = tt * C::BN;
  f32x16 acc[C::TM][C::TN];
  mfma_mainloop<C>(W + (int64_t)v0 * d, d, cend - v0, h + (int64_t)(r0 + t0) * d, d, R - t0, d,
                   reinterpret_cast<bf16_t*>(smem), acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  float* red = reinterpret_cast<float*>(smem);  // [WGM][BN]
  const int vb = v0 + wm * C::WTM;              // vocab id of this wave's first tile row
  const bool full = v0 + C::BM <= cend;         // no tile row past the chunk
  constexpr float kLog2e = 1.4426950408889634f;
  constexpr float kOverSum = 6.2351491e27f;  // e^64
  bool over = false;
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    const int tl = wn * C::WTN + j * 32 + (lane & 31);
    const int t = t0 + tl;
    const bool tok = t < R;
    float ref = 0.0f;
    int y = -1;
    if (tok) {
      ref = label_logit[r0 + t];
      y = labels[r0 + t];
    }
    const float nref = -ref * kLog2e;
    const int ylane = y - vb - 4 * (lane >> 5);
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
      // Register r holds vocab row 8 (r/4) + 4 (lane/32) + r%4 of the 32-row MFMA tile. The
      // per-element label and range tests run only when some lane's label lies in this MFMA
      // tile or the tile crosses the chunk's end.
      const int yl = ylane - i * 32;
      const bool mine = yl >= 0 && yl < 32 && (yl & 4) == 0;
      float e[16];
      if (!full || __ballot(mine) != 0) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = vb + i * 32 + mfma_row(r, lane);
          e[r] = (v < cend && v != y) ? __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, nref)) : 0.0f;
        }
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, nref));
      }
      uint32_t pk[8];
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        sum += e[r];
        sum += e[r + 1];
        pk[r >> 1] = pack_bf16x2(e[r], e[r + 1]);
      }
      // Lanes 0-31 hold rows {0-3, 8-11, 16-19, 24-27}, lanes 32-63 the other four groups.
      // Swapping groups {16-19, 24-27} of the low half with {4-7, 12-15} of the high half
      // leaves rows 0-15 in the low lanes and rows 16-31 in the high lanes, in the same
      // register order for both.
      uint32_t P[4] = {pk[0], pk[1], pk[2], pk[3]}, Q[4] = {pk[4], pk[5], pk[6], pk[7]};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const auto sw = __builtin_amdgcn_permlane32_swap(P[k], Q[k], false, false);
        P[k] = sw[0];
        Q[k] = sw[1];
      }
      if (tok) {
        u32x4* dst = reinterpret_cast<u32x4*>(ez + (int64_t)t * ldz + (vb - c0) + i * 32 + (lane >> 5) * 16);
        dst[0] = u32x4{P[0], P[1], Q[0], Q[1]};
        dst[1] = u32x4{P[2], P[3], Q[2], Q[3]};
      }
    }
    // A single e above e^64 makes the lane's sum exceed it; a sum above it from several
    // smaller terms only runs the exact path needlessly.
    over |= sum > kOverSum;
    sum += __shfl_xor(sum, 32, 64);
    if (lane < 32) red[wm * C::BN + tl] = sum;
  }
  if (over) *flag = 1;
  __syncthreads();
  for (int tl = threadIdx.x; tl < C::BN; tl += C::NT) {
    const int t = t0 + tl;
    if (t >= R) continue;
    float sum = red[tl];
#pragma unroll
    for (int w = 1; w < C::WGM; ++w) sum += red[w * C::BN + tl];
    sig_part[(int64_t)(r0 + t) * n_vb + v0 / C::BM] = sum;
  }
}

// Rows [r0, r0 + R) after the last chunk's first GEMM: sigma_t = sum of the vocab-tile
// partials (fixed order), lse_t = r_t + log1p(sigma_t), row loss w_t log1p(sigma_t), and the
// row scales of the dH epilogue. One wave per row.
__global__ __launch_bounds__(256) void ce_row_final_kernel(int r0, int R, const float* __restrict__ sig_part,
                                                           int n_vb, const float* __restrict__ label_logit,
                                                           const float* __restrict__ weights,
                                                           const float* __restrict__ coef,
                                                           float* __restrict__ lse,
                                                           float* __restrict__ rowloss,
                                                           float* __restrict__ sa, float* __restrict__ sb) {
  const int lane = threadIdx.x & 63;
  const int local = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (local >= R) return;
  const int64_t row = (int64_t)r0 + local;
  float sum = 0.0f;
  for (int i = lane; i < n_vb; i += 64) sum += sig_part[row * n_vb + i];
  sum = group_sum<64>(sum);
  if (lane == 0) {
    const float ce = log1pf(sum);
    const float inv = __fdiv_rn(1.0f, 1.0f + sum);
    const float c = coef[row];
    lse[row] = label_logit[row] + ce;
    rowloss[row] = weights[row] * ce;
    sa[row] = c * inv;
    sb[row] = c * (sum * inv);
  }
}

// coef_t = w_t / L_e for every row of the batch's episodes, 256 rows per block.
__global__ __launch_bounds__(256) void ce_coef_kernel(CeEpBatch b, const float* __restrict__ weights,
                                                      float* __restrict__ coef) {
  int ei = 0;
  while (ei + 1 < b.count && b.e[ei + 1].block_begin <= (int)blockIdx.x) ++ei;
  const CeEp E = b.e[ei];
  const int local = ((int)blockIdx.x - E.block_begin) * 256 + threadIdx.x;
  if (local >= E.L) return;
  const int64_t row = E.row0 + local;
  coef[row] = __fdiv_rn(weights[row], (float)E.L);
}

// ------------------------------------------------------------------------------------------
// f32 path: VALU tiles of 64x64, 256 threads with 4x4 outputs each.
// ------------------------------------------------------------------------------------------
constexpr int kVT = 64, kVK = 16;

// acc += A[0:64, 0:K] * op(B): NT reads B as [64 cols, K] (K-contiguous), NN as [K, 64 cols].
template <bool NN>
__device__ __forceinline__ void valu_mainloop(const float* __restrict__ A, int64_t lda, int mval,
                                              const float* __restrict__ B, int64_t ldb, int nval,
                                              int K, int kval_b, float (&acc)[4][4]) {
  __shared__ float As[kVK][kVT + 4];
  __shared__ float Bs[kVK][kVT + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0f;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  for (int k0 = 0; k0 < K; k0 += kVK) {
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
    if (lr < mval && k0 + lk < K) a = *reinterpret_cast<const float4*>(A + (int64_t)lr * lda + k0 + lk);
    As[lk + 0][lr] = a.x; As[lk + 1][lr] = a.y; As[lk + 2][lr] = a.z; As[lk + 3][lr] = a.w;
    if (!NN) {
      float4 b = make_float4(0.f, 0.f, 0.f, 0.f);
      if (lr < nval && k0 + lk < K) b = *reinterpret_cast<const float4*>(B + (int64_t)lr * ldb + k0 + lk);
      Bs[lk + 0][lr] = b.x; Bs[lk + 1][lr] = b.y; Bs[lk + 2][lr] = b.z; Bs[lk + 3][lr] = b.w;
    } else {
      const int kr = tid >> 4, nc = (tid & 15) * 4;
      float4 b = make_float4(0.f, 0.f, 0.f, 0.f);
      if (k0 + kr < kval_b && nc < nval) b = *reinterpret_cast<const float4*>(B + (int64_t)(k0 + kr) * ldb + nc);
      Bs[kr][nc + 0] = b.x; Bs[kr][nc + 1] = b.y; Bs[kr][nc + 2] = b.z; Bs[kr][nc + 3] = b.w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kVK; ++k) {
      float a4[4], b4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a4[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b4[j] = Bs[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a4[i], b4[j], acc[i][j]);
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void ce_fwd_f32_kernel(const float* __restrict__ h,
                                                         const float* __restrict__ W,
                                                         const int32_t* __restrict__ labels, int N,
                                                         int d, int V, int tiles_m,
                                                         float2* __restrict__ partials, int n_vb,
                                                         float* __restrict__ label_logit) {
  const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
  const int m0 = tm * kVT, n0 = tn * kVT;
  float acc[4][4];
  valu_mainloop<false>(h + (int64_t)m0 * d, d, N - m0, W + (int64_t)n0 * d, d, V - n0, d, 0, acc);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    float mx = -INFINITY;
    for (int j = 0; j < 4; ++j)
      if (n0 + tx * 4 + j < V) mx = fmaxf(mx, acc[i][j]);
    mx = group_max<16>(mx);
    float s = 0.0f;
    if (mx != -INFINITY)
      for (int j = 0; j < 4; ++j)
        if (n0 + tx * 4 + j < V) s += expf(acc[i][j] - mx);
    s = group_sum<16>(s);
    if (row < N) {
      if (tx == 0) partials[(int64_t)row * n_vb + tn] = make_float2(mx, s);
      const int y = labels[row];
      for (int j = 0; j < 4; ++j)
        if (n0 + tx * 4 + j == y) label_logit[row] = acc[i][j];
    }
  }
}

__global__ __launch_bounds__(256) void ce_dz_f32_kernel(const float* __restrict__ h,
                                                        const float* __restrict__ W,
                                                        const int32_t* __restrict__ labels,
                                                        const float* __restrict__ lse,
                                                        const float* __restrict__ coef, int r0,
                                                        int R, int d, int c0, int cend, int V,
                                                        int tiles_m, float* __restrict__ dz,
                                                        int ldz) {
  const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
  const int m0 = tm * kVT, n0 = tn * kVT;
  float acc[4][4];
  valu_mainloop<false>(h + (int64_t)(r0 + m0) * d, d, R - m0, W + (int64_t)(c0 + n0) * d, d,
                       cend - (c0 + n0), d, 0, acc);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  for (int i = 0; i < 4; ++i) {
    const int rl = m0 + ty * 4 + i;
    if (rl >= R) continue;
    const int row = r0 + rl;
    const float l = lse[row], c = coef[row];
    const int y = labels[row];
    for (int j = 0; j < 4; ++j) {
      const int cl = n0 + tx * 4 + j, col = c0 + cl;
      float g = 0.0f;
      if (col < V) g = c * (expf(acc[i][j] - l) - (col == y ? 1.0f : 0.0f));
      dz[(int64_t)rl * ldz + cl] = g;
    }
  }
}

__global__ __launch_bounds__(256) void ce_dh_f32_kernel(const float* __restrict__ dz, int ldz,
                                                        const float* __restrict__ W, int r0, int R,
                                                        int d, int c0, int K, int kval,
                                                        int tiles_m, float* __restrict__ grad,
                                                        int first) {
  const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
  const int m0 = tm * kVT, n0 = tn * kVT;
  float acc[4][4];
  valu_mainloop<true>(dz + (int64_t)m0 * ldz, ldz, R - m0, W + (int64_t)c0 * d + n0, d, d - n0, K,
                      kval, acc);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  for (int i = 0; i < 4; ++i) {
    const int rl = m0 + ty * 4 + i;
    if (rl >= R) continue;
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= d) continue;
      const int64_t o = (int64_t)(r0 + rl) * d + col;
      grad[o] = first ? acc[i][j] : grad[o] + acc[i][j];
    }
  }
}

// ------------------------------------------------------------------------------------------
// Row and episode reductions, LM-head transpose.
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ void ce_row_reduce_body(
    CeEpBatch b, const float2* __restrict__ partials, int n_vb,
    const float* __restrict__ label_logit, const float* __restrict__ weights,
    float* __restrict__ lse, float* __restrict__ coef, float* __restrict__ rowloss) {
  int ei = 0;
  while (ei + 1 < b.count && b.e[ei + 1].block_begin <= (int)blockIdx.x) ++ei;
  const CeEp E = b.e[ei];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int local = ((int)blockIdx.x - E.block_begin) * 4 + wave;
  if (local >= E.L) return;
  const int64_t row = E.row0 + local;
  float m = -INFINITY, s = 0.0f;
  for (int i = lane; i < n_vb; i += 64) {
    const float2 p = partials[row * n_vb + i];
    lse_merge(m, s, p.x, p.y);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(s, o, 64);
    lse_merge(m, s, m2, s2);
  }
  if (lane == 0) {
    const float l = m + logf(s);
    const float w = weights[row];
    lse[row] = l;
    coef[row] = __fdiv_rn(w, (float)E.L);
    rowloss[row] = w * (l - label_logit[row]);
  }
}

__global__ __launch_bounds__(256) void ce_row_reduce_kernel(
    CeEpBatch b, const float2* __restrict__ partials, int n_vb,
    const float* __restrict__ label_logit, const float* __restrict__ weights,
    float* __restrict__ lse, float* __restrict__ coef, float* __restrict__ rowloss) {
  ce_row_reduce_body(b, partials, n_vb, label_logit, weights, lse, coef, rowloss);
}

// The same kernel launched by the overflow guard: returns at once unless *gate != 0.
__global__ __launch_bounds__(256) void ce_guard_row_reduce_kernel(
    CeEpBatch b, const float2* __restrict__ partials, int n_vb,
    const float* __restrict__ label_logit, const float* __restrict__ weights,
    float* __restrict__ lse, float* __restrict__ coef, float* __restrict__ rowloss,
    const int* __restrict__ gate) {
  if (*gate == 0) return;
  ce_row_reduce_body(b, partials, n_vb, label_logit, weights, lse, coef, rowloss);
}

// One 1024-thread workgroup per episode: every thread sums its rows in order (loads issued
// eight at a time), then the waves' sums meet in a fixed order.
constexpr int kLossThreads = 1024;
__device__ __forceinline__ void ce_loss_body(
    CeEpBatch b, const float* __restrict__ rowloss, float* __restrict__ loss) {
  const CeEp E = b.e[blockIdx.x];
  double acc = 0.0;
#pragma unroll 8
  for (int i = threadIdx.x; i < E.L; i += kLossThreads) acc += (double)rowloss[E.row0 + i];
  acc = wave_sum_f64(acc);
  constexpr int kWaves = kLossThreads / 64;
  __shared__ double part[kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int w = 0; w < kWaves; ++w) t += part[w];
    loss[b.first + blockIdx.x] = E.L > 0 ? (float)(t / (double)E.L) : 0.0f;
  }
}

__global__ __launch_bounds__(kLossThreads) void ce_loss_kernel(
    CeEpBatch b, const float* __restrict__ rowloss, float* __restrict__ loss) {
  ce_loss_body(b, rowloss, loss);
}

// The same kernel launched by the overflow guard: returns at once unless *gate != 0.
__global__ __launch_bounds__(kLossThreads) void ce_guard_loss_kernel(
    CeEpBatch b, const float* __restrict__ rowloss, float* __restrict__ loss,
    const int* __restrict__ gate) {
  if (*gate == 0) return;
  ce_loss_body(b, rowloss, loss);
}

// W [V, d] -> WT [d, Vp] in 64 x 64 tiles: 16-byte global reads along d, 16-byte global writes
// along V, through an LDS tile whose padded pitch (66) keeps the column reads conflict-free.
__global__ __launch_bounds__(256) void ce_head_transpose_kernel(const bf16_t* __restrict__ W, int V,
                                                                int d, int Vp,
                                                                bf16_t* __restrict__ WT) {
  constexpr int P = 66;
  __shared__ __align__(16) bf16_t t[64 * P];
  const int v0 = blockIdx.x * 64, j0 = blockIdx.y * 64;
  const int r = threadIdx.x >> 2, c = threadIdx.x & 3;  // row r, 16 columns from 16c
  {
    const int v = v0 + r, j = j0 + 16 * c;
    u32x4 x0 = u32x4{0u, 0u, 0u, 0u}, x1 = u32x4{0u, 0u, 0u, 0u};
    if (v < V && j < d) {
      const u32x4* src = reinterpret_cast<const u32x4*>(W + (int64_t)v * d + j);
      x0 = src[0];
      if (j + 8 < d) x1 = src[1];
    }
    uint32_t* dst = reinterpret_cast<uint32_t*>(t + r * P + 16 * c);  // 4-byte aligned: P even
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      dst[e] = x0[e];
      dst[4 + e] = x1[e];
    }
  }
  __syncthreads();
  const int j = j0 + r, v = v0 + 16 * c;  // output row j, 16 vocab entries from v
  if (j < d && v < Vp) {
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      w[e] = (uint32_t)t[(16 * c + 2 * e) * P + r] | ((uint32_t)t[(16 * c + 2 * e + 1) * P + r] << 16);
    u32x4* out = reinterpret_cast<u32x4*>(WT + (int64_t)j * Vp + v);
    out[0] = u32x4{w[0], w[1], w[2], w[3]};
    out[1] = u32x4{w[4], w[5], w[6], w[7]};
  }
}

// ------------------------------------------------------------------------------------------
// Launchers
// ------------------------------------------------------------------------------------------
template <class Kern>
static hipError_t allow_big_lds(Kern k) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                             hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
}

template <class C>
static hipError_t fwd_bf16(const bf16_t* h, const bf16_t* W, int N, int d, int V, float2* partials,
                           int n_vb, const int* gate, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = allow_big_lds(ce_fwd_bf16_kernel<C>);
    if (e == hipSuccess) e = allow_big_lds(ce_guard_fwd_bf16_kernel<C>);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int tv = (V + C::BM - 1) / C::BM, tt = (N + C::BN - 1) / C::BN;
  KernelTimer t(gate ? K_CE_GUARD : K_CE_FWD, s);
  if (gate)
    hipLaunchKernelGGL(ce_guard_fwd_bf16_kernel<C>, dim3(tv * tt), dim3(C::NT), C::LDS, s, h, W, N, d, V,
                       tv, tt, partials, n_vb, gate);
  else
    hipLaunchKernelGGL(ce_fwd_bf16_kernel<C>, dim3(tv * tt), dim3(C::NT), C::LDS, s, h, W, N, d, V, tv,
                       tt, partials, n_vb);
  return hipGetLastError();
}

hipError_t launch_ce_fwd(int dtype, CeGemmShape t, const void* h, const void* W,
                         const int32_t* labels, int N, int d, int V, float2* partials, int n_vb,
                         float* label_logit, const int* gate, hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (dtype == 1) {
    const bf16_t* hb = static_cast<const bf16_t*>(h);
    const bf16_t* Wb = static_cast<const bf16_t*>(W);
    if (t.bm == 256) return fwd_bf16<CfgBig>(hb, Wb, N, d, V, partials, n_vb, gate, s);
    return fwd_bf16<CfgSmall>(hb, Wb, N, d, V, partials, n_vb, gate, s);
  }
  const int tm = (N + kVT - 1) / kVT, tn = (V + kVT - 1) / kVT;
  KernelTimer tt(K_CE_FWD, s);
  hipLaunchKernelGGL(ce_fwd_f32_kernel, dim3(tm * tn), dim3(256), 0, s,
                     static_cast<const float*>(h), static_cast<const float*>(W), labels, N, d, V, tm,
                     partials, n_vb, label_logit);
  return hipGetLastError();
}

hipError_t launch_ce_label(const void* h, const void* W, const int32_t* labels, int N, int d, int V,
                           float* label_logit, int* flag, hipStream_t s) {
  if (N == 0) return hipSuccess;
  KernelTimer t(K_CE_LABEL, s);
  hipLaunchKernelGGL(ce_label_logit_bf16_kernel, dim3((N + 3) / 4), dim3(256), 0, s,
                     static_cast<const bf16_t*>(h), static_cast<const bf16_t*>(W), labels, N, d, V,
                     label_logit, flag);
  return hipGetLastError();
}

hipError_t launch_ce_row_reduce(const CeEpBatch& b, int total_blocks, const float2* partials,
                                int n_vb, const float* label_logit, const float* weights,
                                float* lse, float* coef, float* rowloss, const int* gate,
                                hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  KernelTimer t(gate ? K_CE_GUARD : K_CE_ROW_REDUCE, s);
  if (gate)
    hipLaunchKernelGGL(ce_guard_row_reduce_kernel, dim3(total_blocks), dim3(256), 0, s, b, partials, n_vb,
                       label_logit, weights, lse, coef, rowloss, gate);
  else
    hipLaunchKernelGGL(ce_row_reduce_kernel, dim3(total_blocks), dim3(256), 0, s, b, partials, n_vb,
                       label_logit, weights, lse, coef, rowloss);
  return hipGetLastError();
}

hipError_t launch_ce_loss(const CeEpBatch& b, const float* rowloss, float* loss, const int* gate,
                          hipStream_t s) {
  if (b.count <= 0) return hipSuccess;
  KernelTimer t(gate ? K_CE_GUARD : K_CE_LOSS, s);
  if (gate)
    hipLaunchKernelGGL(ce_guard_loss_kernel, dim3(b.count), dim3(kLossThreads), 0, s, b, rowloss, loss, gate);
  else
    hipLaunchKernelGGL(ce_loss_kernel, dim3(b.count), dim3(kLossThreads), 0, s, b, rowloss, loss);
  return hipGetLastError();
}

hipError_t launch_ce_coef(const CeEpBatch& b, int total_blocks, const float* weights, float* coef,
                          hipStream_t s) {
  if (total_blocks <= 0) return hipSuccess;
  KernelTimer t(K_CE_ROW_REDUCE, s);
  hipLaunchKernelGGL(ce_coef_kernel, dim3(total_blocks), dim3(256), 0, s, b, weights, coef);
  return hipGetLastError();
}

hipError_t launch_ce_head_transpose(const void* W, int V, int d, int Vp, void* WT, hipStream_t s) {
  KernelTimer t(K_CE_HEAD_T, s);
  hipLaunchKernelGGL(ce_head_transpose_kernel, dim3((Vp + 63) / 64, (d + 63) / 64), dim3(256), 0, s,
                     static_cast<const bf16_t*>(W), V, d, Vp, static_cast<bf16_t*>(WT));
  return hipGetLastError();
}

template <class C>
static hipError_t logit_exp_bf16(const bf16_t* h, const bf16_t* W, const int32_t* labels,
                                 const float* label_logit, int r0, int R, int d, int c0, int Vc, int V,
                                 float* sig_part, int n_vb, bf16_t* ez, int ldz, int* flag,
                                 hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = allow_big_lds(ce_logit_exp_bf16_kernel<C>);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int tv = (Vc + C::BM - 1) / C::BM, tt = (R + C::BN - 1) / C::BN;
  const int cend = min(c0 + Vc, V);
  KernelTimer t(K_CE_LOGIT_EXP, s);
  hipLaunchKernelGGL(ce_logit_exp_bf16_kernel<C>, dim3(tv * tt), dim3(C::NT), C::LDS, s, h, W, labels,
                     label_logit, r0, R, d, c0, cend, tv, tt, sig_part, n_vb, ez, ldz, flag);
  return hipGetLastError();
}

hipError_t launch_ce_logit_exp(CeGemmShape t, const void* h, const void* W, const int32_t* labels,
                               const float* label_logit, int r0, int R, int d, int c0, int Vc, int V,
                               float* sig_part, int n_vb, void* ez, int ldz, int* flag, hipStream_t s) {
  if (R == 0) return hipSuccess;
  const bf16_t* hb = static_cast<const bf16_t*>(h);
  const bf16_t* Wb = static_cast<const bf16_t*>(W);
  bf16_t* z = static_cast<bf16_t*>(ez);
  if (t.bm == 256)
    return logit_exp_bf16<CfgBig>(hb, Wb, labels, label_logit, r0, R, d, c0, Vc, V, sig_part, n_vb, z, ldz,
                                  flag, s);
  return logit_exp_bf16<CfgSmall>(hb, Wb, labels, label_logit, r0, R, d, c0, Vc, V, sig_part, n_vb, z, ldz,
                                  flag, s);
}

hipError_t launch_ce_row_final(int r0, int R, const float* sig_part, int n_vb, const float* label_logit,
                               const float* weights, const float* coef, float* lse, float* rowloss,
                               float* sa, float* sb, hipStream_t s) {
  if (R == 0) return hipSuccess;
  KernelTimer t(K_CE_ROW_REDUCE, s);
  hipLaunchKernelGGL(ce_row_final_kernel, dim3((R + 3) / 4), dim3(256), 0, s, r0, R, sig_part, n_vb,
                     label_logit, weights, coef, lse, rowloss, sa, sb);
  return hipGetLastError();
}

template <class C>
static hipError_t dz_bf16(const bf16_t* h, const bf16_t* W, const int32_t* labels, const float* lse,
                          const float* coef, int r0, int R, int d, int c0, int Vc, int V, bf16_t* dz,
                          int ldz, const int* gate, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = allow_big_lds(ce_dz_bf16_kernel<C>);
    if (e == hipSuccess) e = allow_big_lds(ce_guard_dz_bf16_kernel<C>);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int tm = (R + C::BM - 1) / C::BM, tn = (Vc + C::BN - 1) / C::BN;
  const int cend = min(c0 + Vc, V);
  KernelTimer t(gate ? K_CE_GUARD : K_CE_BWD_DZ, s);
  if (gate)
    hipLaunchKernelGGL(ce_guard_dz_bf16_kernel<C>, dim3(tm * tn), dim3(C::NT), C::LDS, s, h, W, labels, lse,
                       coef, r0, R, d, c0, cend, V, tm, tn, dz, ldz, gate);
  else
    hipLaunchKernelGGL(ce_dz_bf16_kernel<C>, dim3(tm * tn), dim3(C::NT), C::LDS, s, h, W, labels, lse,
                       coef, r0, R, d, c0, cend, V, tm, tn, dz, ldz);
  return hipGetLastError();
}

hipError_t launch_ce_bwd_dz(int dtype, CeGemmShape t, const void* h, const void* W,
                            const int32_t* labels, const float* lse, const float* coef, int r0,
                            int R, int d, int c0, int Vc, int V, void* dz, int ldz, const int* gate,
                            hipStream_t s) {
  if (R == 0) return hipSuccess;
  if (dtype == 1) {
    const bf16_t* hb = static_cast<const bf16_t*>(h);
    const bf16_t* Wb = static_cast<const bf16_t*>(W);
    bf16_t* z = static_cast<bf16_t*>(dz);
    if (t.bm == 256) return dz_bf16<CfgBig>(hb, Wb, labels, lse, coef, r0, R, d, c0, Vc, V, z, ldz, gate, s);
    return dz_bf16<CfgSmall>(hb, Wb, labels, lse, coef, r0, R, d, c0, Vc, V, z, ldz, gate, s);
  }
  const int tm = (R + kVT - 1) / kVT, tn = (Vc + kVT - 1) / kVT;
  const int cend = min(c0 + Vc, V);
  KernelTimer tt(K_CE_BWD_DZ, s);
  hipLaunchKernelGGL(ce_dz_f32_kernel, dim3(tm * tn), dim3(256), 0, s, static_cast<const float*>(h),
                     static_cast<const float*>(W), labels, lse, coef, r0, R, d, c0, cend, V, tm,
                     static_cast<float*>(dz), ldz);
  return hipGetLastError();
}

template <class C>
static hipError_t dh_bf16(const bf16_t* dz, int ldz, const bf16_t* WT, int Vp, int r0, int R, int d,
                          int c0, int K, float* acc, bf16_t* grad, bool first, bool last,
                          const CeRowScale& rs, const bf16_t* W, int V, const int* gate, hipStream_t s) {
  static bool attr = false;
  if (!attr) {
    hipError_t e = allow_big_lds(ce_dh_bf16_kernel<C>);
    if (e == hipSuccess) e = allow_big_lds(ce_guard_dh_bf16_kernel<C>);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const int tm = (d + C::BM - 1) / C::BM, tn = (R + C::BN - 1) / C::BN;  // transposed tiles
  KernelTimer t(gate ? K_CE_GUARD : K_CE_BWD_DH, s);
  if (gate)
    hipLaunchKernelGGL(ce_guard_dh_bf16_kernel<C>, dim3(tm * tn), dim3(C::NT), C::LDS, s, dz, ldz, WT, Vp,
                       r0, R, d, c0, K, tm, tn, acc, grad, first ? 1 : 0, last ? 1 : 0, rs.sa, rs.sb,
                       rs.labels, W, V, gate);
  else
    hipLaunchKernelGGL(ce_dh_bf16_kernel<C>, dim3(tm * tn), dim3(C::NT), C::LDS, s, dz, ldz, WT, Vp, r0,
                       R, d, c0, K, tm, tn, acc, grad, first ? 1 : 0, last ? 1 : 0, rs.sa, rs.sb,
                       rs.labels, W, V);
  return hipGetLastError();
}

hipError_t launch_ce_bwd_dh(int dtype, CeGemmShape t, const void* dz, int ldz, const void* W,
                            const void* WT, int Vp, int r0, int R, int d, int c0, int K, int V,
                            float* acc, void* grad, bool first, bool last, const CeRowScale& rs,
                            const int* gate, hipStream_t s) {
  if (R == 0) return hipSuccess;
  if (dtype == 1) {
    const bf16_t* z = static_cast<const bf16_t*>(dz);
    const bf16_t* wt = static_cast<const bf16_t*>(WT);
    const bf16_t* w = static_cast<const bf16_t*>(W);
    bf16_t* g = static_cast<bf16_t*>(grad);
    if (t.bm == 256) return dh_bf16<CfgBig>(z, ldz, wt, Vp, r0, R, d, c0, K, acc, g, first, last, rs, w, V, gate, s);
    return dh_bf16<CfgSmall>(z, ldz, wt, Vp, r0, R, d, c0, K, acc, g, first, last, rs, w, V, gate, s);
  }
  const int tm = (R + kVT - 1) / kVT, tn = (d + kVT - 1) / kVT;
  KernelTimer tt(K_CE_BWD_DH, s);
  hipLaunchKernelGGL(ce_dh_f32_kernel, dim3(tm * tn), dim3(256), 0, s, static_cast<const float*>(dz),
                     ldz, static_cast<const float*>(W), r0, R, d, c0, K, V - c0, tm,
                     static_cast<float*>(grad), first ? 1 : 0);
  return hipGetLastError();
}

}  // namespace attt
