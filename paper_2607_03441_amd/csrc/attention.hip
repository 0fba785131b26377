// Backward of one adapted attention block (the step before the LoRA gradient: dY_q, dY_k, dY_v
// are the adapter's upstream gradients; Sec. 3.1, Appendix C). Causal attention with grouped
// key/value heads, per episode; head dimension 128; bf16 inputs and outputs, float32
// accumulation. With S = scale Q K^T, P = softmax(S) over the allowed keys, O = P V:
//   D = rowsum(dO * O),  dP = dO V^T,  dS = P * (dP - D),
//   dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO.
// Three kernels, each recomputing S from Q and K on v_mfma_f32_16x16x32_bf16 over blocks of 64
// keys, 256 threads (four waves of 16 rows; 32 query rows in the statistics kernel), blocks in
// the causal order with the longest rows first, the next block's global loads in flight while
// the current one computes:
//   attn_fwd_stats_kernel  per (query head, 128-query block): lse and D (online softmax; D as
//                          the softmax-weighted sum of dP = dO V^T, so O is never formed)
//   attn_dkdv_kernel       per (key/value head, 64-key block): dK and dV accumulated in
//                          registers over every query head of the group and every later query
//                          block, in a fixed order (no atomics)
//   attn_dq_kernel         per (query head, 64-query block): dQ over the allowed key blocks
// The operand that stays in a wave (its 16 queries, or its 16 keys) is held in registers as
// the B operand of the score products, so each lane ends up with 16 scores of its own row. The
// probabilities (or dS) of that row then enter the second product (P^T dO, dS^T Q, dS K)
// directly as the A operand: the contraction index is the one the lane's registers run over,
// in the order they hold it, and the B operand is read in the same order from the row-major LDS
// tile with transposing reads (ds_read_tr16_b64). Every block goes to LDS once, row-major, with
// 16-byte stores, into one of two buffers (one barrier per block). Blocks strictly below the
// diagonal skip the causal and ragged-row masks.
// P and dS enter their second products as bf16 pairs hi + lo (two MFMA passes, about 16
// significant bits): those sums mix signs (dS even sums to zero over each row), and a single
// bf16 rounding of P or dS would show in their small elements. The final bf16 rounding of the
// outputs is then the main error.
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace attt {

namespace {
constexpr int DH = 128;     // head dimension
constexpr int BLK = 64;     // query / key rows per block
constexpr int SBLK = 128;   // query rows per block of the statistics kernel
constexpr int PR = DH + 8;  // LDS pitch of a [64][128] tile (bf16): 272 B, conflict-free b128 reads
constexpr float kLog2e = 1.4426950408889634f;

// LDS: two buffers, so that the next block is stored while the current one is read and a step
// needs one barrier. A buffer of the per-query kernels holds the K and V tiles; one of the
// per-key kernel holds the Q and dO tiles, then lse and D of the block's 64 queries.
constexpr int kTileBytes = BLK * PR * 2;
constexpr int kKvBuf = 2 * kTileBytes;
constexpr int kQoBuf = 2 * kTileBytes + 2 * BLK * 4;

__device__ __forceinline__ bf16_t* kv_tile(uint8_t* smem, int buf, int t) {
  return reinterpret_cast<bf16_t*>(smem + buf * kKvBuf + t * kTileBytes);
}
__device__ __forceinline__ bf16_t* qo_tile(uint8_t* smem, int buf, int t) {
  return reinterpret_cast<bf16_t*>(smem + buf * kQoBuf + t * kTileBytes);
}
__device__ __forceinline__ float* qo_stats(uint8_t* smem, int buf) {  // lse [64], then D [64]
  return reinterpret_cast<float*>(smem + buf * kQoBuf + 2 * kTileBytes);
}

__device__ __forceinline__ bf16_t f2bf(float x) { return (bf16_t)(pack_bf16x2(x, 0.0f) & 0xFFFFu); }

// The block a workgroup works on: episode, head, block index. Workgroups start in launch
// order, so the long causal rows go first: the last query blocks for the per-query kernels
// (`late_first`), the first key blocks for the per-key kernel.
__device__ __forceinline__ void attn_locate(const AttnBatch& b, int heads, bool late_first, int& ei, int& head,
                                            int& blk) {
  ei = 0;
  while (ei + 1 < b.count && b.e[ei + 1].wg_begin <= (int)blockIdx.x) ++ei;
  const int local = (int)blockIdx.x - b.e[ei].wg_begin;
  const int nb = b.e[ei].blocks;
  head = local % heads;
  blk = late_first ? nb - 1 - local / heads : local / heads;
}

}  // namespace

// This wave's 16 keys as MFMA B operands over the head dimension: lane (l16, q4) holds key
// `key` (its own) at columns 32 s + 8 q4 .. +7 for s = 0..3. Keys at or past nvalid read as zero.
__device__ __forceinline__ void load_key_frags(bf16x8 (&f)[4], const bf16_t* src, int64_t stride, int key,
                                               int nvalid, int q4) {
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (key < nvalid) v = *reinterpret_cast<const u32x4*>(src + (int64_t)key * stride + 32 * s + 8 * q4);
    f[s] = __builtin_bit_cast(bf16x8, v);
  }
}

// Rows [0, BLK) of a [rows][DH] block, staged in LDS row-major (pitch PR). Thread tid takes rows
// 4 (tid / 16) .. +3 and columns 8 (tid % 16) .. +7: fetch_block issues its four 16-byte loads
// (rows >= nvalid read as zero), store_block writes them with four 16-byte stores.
// The loads go through one buffer descriptor over the block's valid rows (base and range in
// scalar registers, 32-bit offsets per lane): rows at or past nvalid fall outside its range and
// read as zero. A 64-row block spans less than 2^30 bytes (heads < 2^16, checked on the host).
__device__ __forceinline__ void fetch_block(u32x4 (&v)[4], const bf16_t* src, int64_t stride, int nvalid, int tid) {
  const int r0 = (tid >> 4) * 4, c0 = (tid & 15) * 8;
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(src, nvalid > 0 ? (int)(((int64_t)(nvalid - 1) * stride + DH) * 2) : 0);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    v[i] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (uint32_t)(((int64_t)(r0 + i) * stride + c0) * 2), 0, 0));
}

__device__ __forceinline__ void store_block(const u32x4 (&v)[4], bf16_t* dst, int tid) {
  const int r0 = (tid >> 4) * 4, c0 = (tid & 15) * 8;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(dst + (r0 + i) * PR + c0) = v[i];
}

// hi = RN(x), lo = RN(x - hi) of the eight values of an MFMA operand, as bf16x8 pairs.
__device__ __forceinline__ void split_frag(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
  u32x4 h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
    l[i] = pack_bf16x2(x[2 * i] - bf16_bits_to_f32(h[i] & 0xFFFFu), x[2 * i + 1] - bf16_bits_to_f32(h[i] >> 16));
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

// B operand of the second products over the 32 rows (queries, or keys) of chunk u, from a
// row-major [64][DH] tile (pitch PR) through transposing LDS reads: lane (l16, q4) receives
// column c0 + l16 at rows 32 u + 4 q4 .. +3 and 32 u + 16 + 4 q4 .. +3, the order in which the
// P / dS fragments hold them. ds_read_tr16_b64 hands, within each group of 16 lanes, lane i the
// element i mod 4 of lanes 4e + i/4 (e = 0..3), so lane 4e + c of group q4 addresses row
// 32 u + 4 q4 + e (then 16 rows further) at columns c0 + 4c .. +3.
__device__ __forceinline__ bf16x8 trfrag(const bf16_t* R, int c0, int u, int lane) {
  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) v4s* lds_v4s;
  const int q4 = lane >> 4, e = (lane >> 2) & 3, c = lane & 3;
  const bf16_t* p = R + (32 * u + 4 * q4 + e) * PR + c0 + 4 * c;
  const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p));
  const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p + 16 * PR));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  return __builtin_bit_cast(bf16x8, u32x4{a.x, a.y, b.x, b.y});
}

// lse and D = rowsum(dO * O) of one (query head, 128-query block). Wave w owns queries 32 w ..
// 32 w + 31 as two tiles of 16; their Q and dO fragments stay in registers. Per key block: S^T =
// K Q^T and dP^T = V dO^T with the keys on the MFMA rows, each K and V fragment read from LDS once
// for both tiles, so each lane holds 16 scores of each of its two queries and the online softmax
// of a query is a reduction over the lane's registers and its three partner lanes (lanes l,
// l + 16, l + 32, l + 48 hold the same queries). O = P V is never formed: since
// O = sum_k P_k V_k, D = sum_k P_k (dO . V_k) = sum_k P_k dP_k, so each lane keeps, beside the
// running softmax sum, the running sum of p dP over its keys, both rescaled by the same factor
// when the running max grows; the four partial sums of a query are added at the end.
__global__ __launch_bounds__(256, 2) void attn_fwd_stats_kernel(AttnArgs a, AttnBatch b) {
  int ei, h, qb;
  attn_locate(b, a.heads, true, ei, h, qb);
  const AttnEp E = b.e[ei];
  const int kh = h / (a.heads / a.kv_heads);
  const int q0 = qb * SBLK, nq = min(SBLK, E.L - q0);
  extern __shared__ __align__(16) uint8_t smem[];  // two buffers of [K tile][V tile], [64][PR] each
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const int64_t qs = (int64_t)a.heads * DH, ks = (int64_t)a.kv_heads * DH;
  bf16x8 qf[2][4], of[2][4];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int qry = 32 * w + 16 * c + l16;
    load_key_frags(qf[c], a.q + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, qry, nq, q4);
    load_key_frags(of[c], a.dout + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, qry, nq, q4);
  }
  const float sl = a.scale * kLog2e;
  // per query tile: running max (base 2, the same in the query's four lanes), and this lane's
  // running sums of p and of p dP over its keys
  float m[2] = {-INFINITY, -INFINITY}, l[2] = {0.0f, 0.0f}, dacc[2] = {0.0f, 0.0f};
  u32x4 fk[4], fv[4];
  auto fetch = [&](int kb) {
    const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
    fetch_block(fk, a.k + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
    fetch_block(fv, a.v + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
  };
  const int kb_last = (q0 + nq - 1) / BLK;  // the key block of the block's last query
  const int wq0 = q0 + 32 * w;              // this wave's first query
  fetch(0);
  store_block(fk, kv_tile(smem, 0, 0), tid);
  store_block(fv, kv_tile(smem, 0, 1), tid);
  for (int kb = 0; kb <= kb_last; ++kb) {
    const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
    // This block's tiles are stored, and every wave is done with the other buffer.
    __syncthreads();
    if (kb < kb_last) fetch(kb + 1);  // the next key block loads while this one computes
    // A wave whose queries all precede the block has nothing to add (it still takes part in
    // the barriers and the stores).
    if (k0 <= wq0 + 31) {
      const bf16_t* Ks = kv_tile(smem, kb & 1, 0);
      const bf16_t* Vs = kv_tile(smem, kb & 1, 1);
      // S^T[16 tt + 4 q4 + r][query] and dP^T likewise, for both query tiles
      f32x4 st[2][4], dp[2][4];
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) st[c][tt] = f32x4{0, 0, 0, 0}, dp[c][tt] = f32x4{0, 0, 0, 0};
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
          const bf16x8 ak = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(Ks + (16 * tt + l16) * PR + 32 * s4 + 8 * q4));
          const bf16x8 av = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(Vs + (16 * tt + l16) * PR + 32 * s4 + 8 * q4));
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            st[c][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, qf[c][s4], st[c][tt], 0, 0, 0);
            dp[c][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, of[c][s4], dp[c][tt], 0, 0, 0);
          }
        }
      // each K and V fragment pair is read just ahead of its four products, which bounds the
      // registers held by reads in flight
#pragma unroll
      for (int n = 0; n < 16; ++n) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
      }
      // online softmax (base-2 exponent of scale * S) over this block's keys 16 tt + 4 q4 + r.
      // A whole key block that ends at or before the wave's first query is entirely allowed:
      // no mask there.
      auto softmax = [&](auto masked) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int qry = 32 * w + 16 * c + l16;
          float mx = -INFINITY, sum = 0.0f, dsum = 0.0f;
#pragma unroll
          for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int kl = 16 * tt + 4 * q4 + r;
              float v = st[c][tt][r] * sl;
              if constexpr (decltype(masked)::value) v = (k0 + kl <= q0 + qry && kl < nk) ? v : -INFINITY;
              st[c][tt][r] = v;
              mx = fmaxf(mx, v);
            }
          mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
          mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
          const float mn = fmaxf(m[c], mx);
#pragma unroll
          for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              float p = __builtin_amdgcn_exp2f(st[c][tt][r] - mn);
              if constexpr (decltype(masked)::value) p = (st[c][tt][r] == -INFINITY) ? 0.0f : p;
              sum += p;
              dsum += p * dp[c][tt][r];
            }
          const float alpha = (m[c] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m[c] - mn);
          l[c] = l[c] * alpha + sum;
          dacc[c] = dacc[c] * alpha + dsum;
          m[c] = mn;
        }
      };
      if (k0 + BLK - 1 <= wq0 && nk == BLK)
        softmax(std::false_type{});
      else
        softmax(std::true_type{});
    }
    if (kb < kb_last) {
      store_block(fk, kv_tile(smem, (kb + 1) & 1, 0), tid);
      store_block(fv, kv_tile(smem, (kb + 1) & 1, 1), tid);
    }
  }
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int qry = 32 * w + 16 * c + l16;
    float lc = l[c], dc = dacc[c];
    lc += __shfl_xor(lc, 16, 64);
    lc += __shfl_xor(lc, 32, 64);
    dc += __shfl_xor(dc, 16, 64);
    dc += __shfl_xor(dc, 32, 64);
    if (q4 == 0 && qry < nq) {
      const int64_t t = (int64_t)h * a.N + E.row0 + q0 + qry;
      a.lse[t] = m[c] / kLog2e + logf(lc);
      a.dsum[t] = dc / lc;
    }
  }
}

// dK, dV of one (key/value head, 64-key block). Wave w owns keys 16 w .. 16 w + 15; their K and
// V fragments stay in registers. Per query block: S = Q K^T and dP = dO V^T with the queries on
// the MFMA rows (four tiles of 16) and this wave's keys on the columns, so each lane holds 16
// (query, key) values of its own key. P and dS = P (dP - D) then feed dV += P^T dO and
// dK += dS^T Q straight from those registers as the A operand: the contraction runs over the
// queries, and the 8 values a lane holds per 32-query chunk (tile rows 4 q4 .. +3 of two tiles)
// are its k slots; the B operand reads the transposed dO and Q tiles in the same query order.
__global__ __launch_bounds__(256, 2) void attn_dkdv_kernel(AttnArgs a, AttnBatch b) {
  int ei, kh, kb;
  attn_locate(b, a.kv_heads, false, ei, kh, kb);
  const AttnEp E = b.e[ei];
  const int g = a.heads / a.kv_heads;
  const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
  extern __shared__ __align__(16) uint8_t smem[];  // two buffers of [Q tile][dO tile][lse][D]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const int key = 16 * w + l16;  // this lane's key in the block
  const int64_t qs = (int64_t)a.heads * DH, ks = (int64_t)a.kv_heads * DH;
  bf16x8 kf[4], vf[4];
  load_key_frags(kf, a.k + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, key, nk, q4);
  load_key_frags(vf, a.v + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, key, nk, q4);
  f32x4 dk[8], dv[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) dk[j] = f32x4{0, 0, 0, 0}, dv[j] = f32x4{0, 0, 0, 0};
  const float sl = a.scale * kLog2e;
  const int nqb = (E.L + BLK - 1) / BLK;
  // (query block, query head) steps: query blocks from the last down to kb, the group's query
  // heads inside. Every workgroup of a key/value head walks the same blocks in the same order
  // (starting at the last, stopping at its own key block), so those running together on an XCD
  // read each Q and dO block from its L2.
  const int steps = g * (nqb - kb);
  u32x4 fq[4], fo[4];
  float fl = INFINITY, fd = 0.0f;
  auto fetch = [&](int i) {
    const int h = kh * g + i % g, q0 = (nqb - 1 - i / g) * BLK, nq = min(BLK, E.L - q0);
    fetch_block(fq, a.q + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
    fetch_block(fo, a.dout + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
    if (tid < BLK) {
      const int64_t t = (int64_t)h * a.N + E.row0 + q0 + tid;
      fl = tid < nq ? a.lse[t] * kLog2e : INFINITY;  // absent rows: P = 0
      fd = tid < nq ? a.dsum[t] : 0.0f;
    }
  };
  auto stage = [&](int buf) {
    store_block(fq, qo_tile(smem, buf, 0), tid);
    store_block(fo, qo_tile(smem, buf, 1), tid);
    if (tid < BLK) qo_stats(smem, buf)[tid] = fl, qo_stats(smem, buf)[BLK + tid] = fd;
  };
  fetch(0);
  stage(0);
  for (int i = 0; i < steps; ++i) {
    const int q0 = (nqb - 1 - i / g) * BLK;
    // This step's tiles are stored, and every wave is done with the other buffer.
    __syncthreads();
    if (i + 1 < steps) fetch(i + 1);  // the next step's blocks load while this one computes
    const bf16_t* Qs = qo_tile(smem, i & 1, 0);
    const bf16_t* dOs = qo_tile(smem, i & 1, 1);
    const float* lse_s = qo_stats(smem, i & 1);
    const float* d_s = lse_s + BLK;
    {
      // S[16 t + 4 q4 + r][key] and dP likewise
      f32x4 st[4], dp[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) st[t] = f32x4{0, 0, 0, 0}, dp[t] = f32x4{0, 0, 0, 0};
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const bf16x8 aq = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(Qs + (16 * t + l16) * PR + 32 * s4 + 8 * q4));
          const bf16x8 ao = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const u32x4*>(dOs + (16 * t + l16) * PR + 32 * s4 + 8 * q4));
          st[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, kf[s4], st[t], 0, 0, 0);
          dp[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ao, vf[s4], dp[t], 0, 0, 0);
        }
      // P and dS of this lane's 16 (query, key) pairs, in fragment order: chunk u, slot i is
      // query 32 u + 4 q4 + i (i < 4) or 32 u + 16 + 4 q4 + i - 4. A query block after the key
      // block sees every key, and the key block is then not the last, so it is whole: no mask.
      float pv[2][8], dsv[2][8];
      auto probs = [&](auto masked) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const f32x4 ls = *reinterpret_cast<const f32x4*>(lse_s + 16 * t + 4 * q4);
          const f32x4 dd = *reinterpret_cast<const f32x4*>(d_s + 16 * t + 4 * q4);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ql = 16 * t + 4 * q4 + r;
            float p = __builtin_amdgcn_exp2f(st[t][r] * sl - ls[r]);
            if constexpr (decltype(masked)::value) p = (k0 + key <= q0 + ql && key < nk) ? p : 0.0f;
            pv[t >> 1][4 * (t & 1) + r] = p;
            dsv[t >> 1][4 * (t & 1) + r] = p * (dp[t][r] - dd[r]);
          }
        }
      };
      if (q0 > k0)
        probs(std::false_type{});
      else
        probs(std::true_type{});
      bf16x8 ph[2], pl[2], sh[2], slo[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        split_frag(pv[u], ph[u], pl[u]);
        split_frag(dsv[u], sh[u], slo[u]);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const bf16x8 bo = trfrag(dOs, 16 * j, u, lane);
          dv[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[u], bo, dv[j], 0, 0, 0);
          dv[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl[u], bo, dv[j], 0, 0, 0);
          const bf16x8 bq = trfrag(Qs, 16 * j, u, lane);
          dk[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sh[u], bq, dk[j], 0, 0, 0);
          dk[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(slo[u], bq, dk[j], 0, 0, 0);
        }
    }
    if (i + 1 < steps) stage((i + 1) & 1);
  }
  // D of dV / dK tile j: lane (l16, q4), register r -> key 16 w + 4 q4 + r, column 16 j + l16
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int kr = 16 * w + 4 * q4 + r;
    if (kr >= nk) continue;
    bf16_t* dkr = a.dk + ((int64_t)(E.row0 + k0 + kr) * a.kv_heads + kh) * DH;
    bf16_t* dvr = a.dv + ((int64_t)(E.row0 + k0 + kr) * a.kv_heads + kh) * DH;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      dkr[16 * j + l16] = f2bf(dk[j][r] * a.scale);
      dvr[16 * j + l16] = f2bf(dv[j][r]);
    }
  }
}

// dQ of one (query head, 64-query block). Wave w owns queries 16 w .. 16 w + 15; their Q and
// dO fragments stay in registers. Per key block: S^T = K Q^T and dP^T = V dO^T with the keys on
// the MFMA rows and this wave's queries on the columns, so each lane holds 16 (key, query)
// values of its own query; dS then feeds dQ += dS K as the A operand (the contraction runs over
// the keys in the order the lane holds them), with the B operand from the transposed K tile.
__global__ __launch_bounds__(256, 2) void attn_dq_kernel(AttnArgs a, AttnBatch b) {
  int ei, h, qb;
  attn_locate(b, a.heads, true, ei, h, qb);
  const AttnEp E = b.e[ei];
  const int kh = h / (a.heads / a.kv_heads);
  const int q0 = qb * BLK, nq = min(BLK, E.L - q0);
  extern __shared__ __align__(16) uint8_t smem[];  // two buffers of [K tile][V tile], [64][PR] each
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const int qry = 16 * w + l16;  // this lane's query in the block
  const int64_t qs = (int64_t)a.heads * DH, ks = (int64_t)a.kv_heads * DH;
  bf16x8 qf[4], of[4];
  load_key_frags(qf, a.q + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, qry, nq, q4);
  load_key_frags(of, a.dout + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, qry, nq, q4);
  const int64_t t = (int64_t)h * a.N + E.row0 + q0 + qry;
  const float ls = qry < nq ? a.lse[t] * kLog2e : INFINITY;  // absent queries: P = 0
  const float dd = qry < nq ? a.dsum[t] : 0.0f;
  f32x4 dq[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) dq[j] = f32x4{0, 0, 0, 0};
  const float sl = a.scale * kLog2e;
  u32x4 fk[4], fv[4];
  auto fetch = [&](int kb) {
    const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
    fetch_block(fk, a.k + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
    fetch_block(fv, a.v + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
  };
  fetch(0);
  store_block(fk, kv_tile(smem, 0, 0), tid);
  store_block(fv, kv_tile(smem, 0, 1), tid);
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
    // This block's tiles are stored, and every wave is done with the other buffer.
    __syncthreads();
    if (kb < qb) fetch(kb + 1);  // the next key block loads while this one computes
    const bf16_t* Ks = kv_tile(smem, kb & 1, 0);
    const bf16_t* Vs = kv_tile(smem, kb & 1, 1);
    // S^T[16 t + 4 q4 + r][query] and dP^T likewise
    f32x4 st[4], dp[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) st[tt] = f32x4{0, 0, 0, 0}, dp[tt] = f32x4{0, 0, 0, 0};
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const bf16x8 ak = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(Ks + (16 * tt + l16) * PR + 32 * s4 + 8 * q4));
        const bf16x8 av = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(Vs + (16 * tt + l16) * PR + 32 * s4 + 8 * q4));
        st[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, qf[s4], st[tt], 0, 0, 0);
        dp[tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, of[s4], dp[tt], 0, 0, 0);
      }
    // dS of this lane's query against 16 keys, in fragment order: chunk u, slot i is key
    // 32 u + 4 q4 + i (i < 4) or 32 u + 16 + 4 q4 + i - 4. A key block before the query block
    // is whole and entirely allowed: no mask there.
    float dsv[2][8];
    auto grad = [&](auto masked) {
#pragma unroll
      for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kl = 16 * tt + 4 * q4 + r;
          float p = __builtin_amdgcn_exp2f(st[tt][r] * sl - ls);
          if constexpr (decltype(masked)::value) p = (k0 + kl <= q0 + qry && kl < nk) ? p : 0.0f;
          dsv[tt >> 1][4 * (tt & 1) + r] = p * (dp[tt][r] - dd);
        }
    };
    if (kb < qb)
      grad(std::false_type{});
    else
      grad(std::true_type{});
    bf16x8 sh[2], slo[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) split_frag(dsv[u], sh[u], slo[u]);
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const bf16x8 bk = trfrag(Ks, 16 * j, u, lane);
        dq[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sh[u], bk, dq[j], 0, 0, 0);
        dq[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(slo[u], bk, dq[j], 0, 0, 0);
      }
    if (kb < qb) {
      store_block(fk, kv_tile(smem, (kb + 1) & 1, 0), tid);
      store_block(fv, kv_tile(smem, (kb + 1) & 1, 1), tid);
    }
  }
  // D of dQ tile j: lane (l16, q4), register r -> query 16 w + 4 q4 + r, column 16 j + l16
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qi = 16 * w + 4 * q4 + r;
    if (qi >= nq) continue;
    bf16_t* dqr = a.dq + ((int64_t)(E.row0 + q0 + qi) * a.heads + h) * DH;
#pragma unroll
    for (int j = 0; j < 8; ++j) dqr[16 * j + l16] = f2bf(dq[j][r] * a.scale);
  }
}

size_t attn_lds_bytes(int kernel) { return 2 * (size_t)(kernel == 1 ? kQoBuf : kKvBuf); }

hipError_t launch_attn(int kernel, const AttnArgs& a, const AttnBatch& b, int wgs, hipStream_t s) {
  if (wgs <= 0) return hipSuccess;
  static bool attr[3] = {false, false, false};
  const void* fns[3] = {(const void*)attn_fwd_stats_kernel, (const void*)attn_dkdv_kernel, (const void*)attn_dq_kernel};
  const size_t lds = attn_lds_bytes(kernel);
  if (!attr[kernel]) {
    hipError_t e = hipFuncSetAttribute(fns[kernel], hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr[kernel] = true;
  }
  KernelTimer t(kernel == 0 ? K_ATTN_FWD : kernel == 1 ? K_ATTN_DKDV : K_ATTN_DQ, s);
  if (kernel == 0) {
    // the statistics kernel works on 128-query blocks: its own block counts and grid
    AttnBatch b2 = b;
    int n = 0;
    for (int i = 0; i < b2.count; ++i) {
      b2.e[i].blocks = (b2.e[i].L + SBLK - 1) / SBLK;
      b2.e[i].wg_begin = n;
      n += b2.e[i].blocks * a.heads;
    }
    if (n > 0) hipLaunchKernelGGL(attn_fwd_stats_kernel, dim3(n), dim3(256), lds, s, a, b2);
  }
  if (kernel == 1) hipLaunchKernelGGL(attn_dkdv_kernel, dim3(wgs), dim3(256), lds, s, a, b);
  if (kernel == 2) hipLaunchKernelGGL(attn_dq_kernel, dim3(wgs), dim3(256), lds, s, a, b);
  return hipGetLastError();
}

}  // namespace attt
