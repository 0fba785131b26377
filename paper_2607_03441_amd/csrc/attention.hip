// Backward of one adapted attention block (the step before the LoRA gradient: dY_q, dY_k, dY_v
// are the adapter's upstream gradients; Sec. 3.1, Appendix C). Causal attention with grouped
// key/value heads, per episode; head dimension 128; bf16 inputs and outputs, float32
// accumulation. With S = scale Q K^T, P = softmax(S) over the allowed keys, O = P V:
//   D = rowsum(dO * O),  dP = dO V^T,  dS = P * (dP - D),
//   dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO.
// Three kernels, each recomputing S from Q and K on v_mfma_f32_16x16x32_bf16 (64 x 64 blocks,
// four waves of 16 rows; operands in LDS rows padded so that fragment reads do not conflict):
//   attn_fwd_stats_kernel  per (query head, 64-query block): lse and D (online softmax; O kept
//                          in float32 registers and contracted with dO, never written)
//   attn_dkdv_kernel       per (key/value head, 64-key block): dK and dV accumulated in
//                          registers over every query head of the group and every later query
//                          block, in a fixed order (no atomics)
//   attn_dq_kernel         per (query head, 64-query block): dQ over the allowed key blocks
// P and dS enter their second products (O = P V for D, dV = P^T dO, dQ = dS K, dK = dS^T Q) as
// bf16 pairs hi + lo (two MFMA passes, about 16 significant bits): those sums mix signs (dS even
// sums to zero over each row), and a single bf16 rounding of P or dS would show in their small
// elements. The final bf16 rounding of the outputs is then the main error.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

namespace {
constexpr int DH = 128;     // head dimension
constexpr int BLK = 64;     // query / key rows per block
constexpr int PR = DH + 8;  // LDS pitch of a [64][128] tile (bf16): 272 B, conflict-free b128 reads
constexpr int PT = BLK + 8; // LDS pitch of a transposed [128][64] tile and of P / dS staging
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ bf16_t f2bf(float x) { return (bf16_t)(pack_bf16x2(x, 0.0f) & 0xFFFFu); }

// rows [0, BLK) of a [rows][DH] bf16 tensor (row stride `stride` elements) into LDS `dst`
// (pitch PR) if given and, if `dstT` is given, transposed into dstT[c][r] (pitch PT). Rows >=
// nvalid read as zero.
__device__ __forceinline__ void load_block(bf16_t* dst, bf16_t* dstT, const bf16_t* src, int64_t stride,
                                           int nvalid, int tid) {
#pragma unroll
  for (int i = 0; i < (BLK * DH / 8) / 256; ++i) {
    const int c = tid + 256 * i;
    const int r = c >> 4, c8 = (c & 15) * 8;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (r < nvalid) v = *reinterpret_cast<const u32x4*>(src + (int64_t)r * stride + c8);
    if (dst) *reinterpret_cast<u32x4*>(dst + r * PR + c8) = v;
    if (dstT) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dstT[(c8 + 2 * e) * PT + r] = (bf16_t)(v[e] & 0xFFFFu);
        dstT[(c8 + 2 * e + 1) * PT + r] = (bf16_t)(v[e] >> 16);
      }
    }
  }
}

// acc[j] += A[row0 + 0..15][0..32*KS) * B[col0 + 16 j + 0..15][0..32*KS)^T, both LDS row-major
// with K contiguous (pitches lda, ldb).
template <int KS, int NJ>
__device__ __forceinline__ void mma_nt(const bf16_t* A, int lda, int row0, const bf16_t* B, int ldb, int col0,
                                       f32x4 (&acc)[NJ], int lane) {
  const int l16 = lane & 15, q4 = lane >> 4;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(A + (row0 + l16) * lda + ks * 32 + q4 * 8));
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const bf16x8 b = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(B + (col0 + 16 * j + l16) * ldb + ks * 32 + q4 * 8));
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
    }
  }
}

// The block a workgroup works on: episode, head, block index.
__device__ __forceinline__ void attn_locate(const AttnBatch& b, int heads, int& ei, int& head, int& blk) {
  ei = 0;
  while (ei + 1 < b.count && b.e[ei + 1].wg_begin <= (int)blockIdx.x) ++ei;
  const int local = (int)blockIdx.x - b.e[ei].wg_begin;
  const int nb = b.e[ei].blocks;
  // long rows of blocks first (causal work grows with the block index)
  head = local % heads;
  blk = nb - 1 - local / heads;
}

}  // namespace

__global__ __launch_bounds__(256) void attn_fwd_stats_kernel(AttnArgs a, AttnBatch b) {
  int ei, h, qb;
  attn_locate(b, a.heads, ei, h, qb);
  const AttnEp E = b.e[ei];
  const int kh = h / (a.heads / a.kv_heads);
  const int q0 = qb * BLK, nq = min(BLK, E.L - q0);
  extern __shared__ __align__(16) uint8_t smem[];
  bf16_t* Qs = reinterpret_cast<bf16_t*>(smem);  // [64][PR]
  bf16_t* Ks = Qs + BLK * PR;                     // [64][PR]
  bf16_t* Vt = Ks + BLK * PR;                     // [128][PT]
  bf16_t* Ps = Vt + DH * PT;                      // [64][PT] P, high part
  bf16_t* Pl = Ps + BLK * PT;                     // low part
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const int64_t qs = (int64_t)a.heads * DH, ks = (int64_t)a.kv_heads * DH;
  load_block(Qs, nullptr, a.q + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
  const float sl = a.scale * kLog2e;
  float m[4], l[4];
  f32x4 o[8];
#pragma unroll
  for (int r = 0; r < 4; ++r) m[r] = -INFINITY, l[r] = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) o[j] = f32x4{0, 0, 0, 0};
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
    __syncthreads();  // previous block's reads of Ks / Vt / Ps are done
    load_block(Ks, nullptr, a.k + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
    load_block(nullptr, Vt, a.v + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
    __syncthreads();
    f32x4 s[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] = f32x4{0, 0, 0, 0};
    mma_nt<DH / 32, 4>(Qs, PR, 16 * w, Ks, PR, 0, s, lane);
    // online softmax over this block (base-2 exponent of scale * S)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int qi = q0 + 16 * w + 4 * q4 + r;
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kj = k0 + 16 * j + l16;
        const float v = (kj <= qi && kj < E.L) ? s[j][r] * sl : -INFINITY;
        s[j][r] = v;
        mx = fmaxf(mx, v);
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      const float mn = fmaxf(m[r], mx);
      const float alpha = (m[r] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m[r] - mn);
      float sum = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p = (s[j][r] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(s[j][r] - mn);
        s[j][r] = p;
        sum += p;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) sum += __shfl_xor(sum, off, 64);
      l[r] = l[r] * alpha + sum;
      m[r] = mn;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j][r] *= alpha;
    }
    // P (bf16) of this wave's rows to LDS (the previous block's reads of Ps ended before the
    // barrier at the top of this block), then O += P V
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bf16_t hi = f2bf(s[j][r]);
        Ps[(16 * w + 4 * q4 + r) * PT + 16 * j + l16] = hi;
        Pl[(16 * w + 4 * q4 + r) * PT + 16 * j + l16] = f2bf(s[j][r] - bf2f(hi));
      }
    __syncthreads();
    mma_nt<BLK / 32, 8>(Ps, PT, 16 * w, Vt, PT, 0, o, lane);
    mma_nt<BLK / 32, 8>(Pl, PT, 16 * w, Vt, PT, 0, o, lane);
  }
  // lse (natural log) and D = rowsum(dO * O) of this wave's 16 rows
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qi = 16 * w + 4 * q4 + r;
    const float inv = l[r] > 0.0f ? 1.0f / l[r] : 0.0f;
    float d = 0.0f;
    if (qi < nq) {
      const bf16_t* dor = a.dout + ((int64_t)(E.row0 + q0 + qi) * a.heads + h) * DH;
#pragma unroll
      for (int j = 0; j < 8; ++j) d += bf2f(dor[16 * j + l16]) * (o[j][r] * inv);
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) d += __shfl_xor(d, off, 64);
    if (l16 == 0 && qi < nq) {
      const int64_t t = (int64_t)h * a.N + E.row0 + q0 + qi;
      a.lse[t] = m[r] / kLog2e + logf(l[r]);
      a.dsum[t] = d;
    }
  }
}

__global__ __launch_bounds__(256) void attn_dkdv_kernel(AttnArgs a, AttnBatch b) {
  int ei, kh, kb;
  attn_locate(b, a.kv_heads, ei, kh, kb);
  const AttnEp E = b.e[ei];
  const int g = a.heads / a.kv_heads;
  const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
  extern __shared__ __align__(16) uint8_t smem[];
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);  // [64][PR]
  bf16_t* Vs = Ks + BLK * PR;
  bf16_t* Qs = Vs + BLK * PR;
  bf16_t* dOs = Qs + BLK * PR;
  bf16_t* Qt = dOs + BLK * PR;                    // [128][PT]
  bf16_t* dOt = Qt + DH * PT;
  bf16_t* PTs = dOt + DH * PT;                    // [64 keys][PT] P^T, high part
  bf16_t* PTl = PTs + BLK * PT;                   // P^T, low part
  bf16_t* dSTs = PTl + BLK * PT;                  // dS^T, high part
  bf16_t* dSTl = dSTs + BLK * PT;                 // dS^T, low part
  float* lse_s = reinterpret_cast<float*>(dSTl + BLK * PT);  // [64]
  float* d_s = lse_s + BLK;                                  // [64]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const int64_t qs = (int64_t)a.heads * DH, ks = (int64_t)a.kv_heads * DH;
  load_block(Ks, nullptr, a.k + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
  load_block(Vs, nullptr, a.v + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
  f32x4 dk[8], dv[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) dk[j] = f32x4{0, 0, 0, 0}, dv[j] = f32x4{0, 0, 0, 0};
  const float sl = a.scale * kLog2e;
  const int nqb = (E.L + BLK - 1) / BLK;
  for (int hh = 0; hh < g; ++hh) {
    const int h = kh * g + hh;
    for (int qb = kb; qb < nqb; ++qb) {
      const int q0 = qb * BLK, nq = min(BLK, E.L - q0);
      __syncthreads();  // previous step's reads are done
      load_block(Qs, Qt, a.q + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
      load_block(dOs, dOt, a.dout + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
      if (tid < BLK) {
        const int64_t t = (int64_t)h * a.N + E.row0 + q0 + tid;
        lse_s[tid] = tid < nq ? a.lse[t] * kLog2e : INFINITY;  // absent rows: P = 0
        d_s[tid] = tid < nq ? a.dsum[t] : 0.0f;
      }
      __syncthreads();
      // S^T and dP^T: this wave's 16 keys x 64 queries
      f32x4 st[4], dpt[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) st[j] = f32x4{0, 0, 0, 0}, dpt[j] = f32x4{0, 0, 0, 0};
      mma_nt<DH / 32, 4>(Ks, PR, 16 * w, Qs, PR, 0, st, lane);
      mma_nt<DH / 32, 4>(Vs, PR, 16 * w, dOs, PR, 0, dpt, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int qc = 16 * j + l16;  // query column
        const float ls = lse_s[qc], dd = d_s[qc];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kr = 16 * w + 4 * q4 + r;  // key row
          const bool ok = (k0 + kr <= q0 + qc) && (kr < nk);
          const float p = ok ? __builtin_amdgcn_exp2f(st[j][r] * sl - ls) : 0.0f;
          const float ds = p * (dpt[j][r] - dd);
          const bf16_t hi = f2bf(ds), phi = f2bf(p);
          PTs[kr * PT + qc] = phi;
          PTl[kr * PT + qc] = f2bf(p - bf2f(phi));
          dSTs[kr * PT + qc] = hi;
          dSTl[kr * PT + qc] = f2bf(ds - bf2f(hi));
        }
      }
      __syncthreads();
      mma_nt<BLK / 32, 8>(PTs, PT, 16 * w, dOt, PT, 0, dv, lane);
      mma_nt<BLK / 32, 8>(PTl, PT, 16 * w, dOt, PT, 0, dv, lane);
      mma_nt<BLK / 32, 8>(dSTs, PT, 16 * w, Qt, PT, 0, dk, lane);
      mma_nt<BLK / 32, 8>(dSTl, PT, 16 * w, Qt, PT, 0, dk, lane);
    }
  }
  // write this wave's 16 keys
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

__global__ __launch_bounds__(256) void attn_dq_kernel(AttnArgs a, AttnBatch b) {
  int ei, h, qb;
  attn_locate(b, a.heads, ei, h, qb);
  const AttnEp E = b.e[ei];
  const int kh = h / (a.heads / a.kv_heads);
  const int q0 = qb * BLK, nq = min(BLK, E.L - q0);
  extern __shared__ __align__(16) uint8_t smem[];
  bf16_t* Qs = reinterpret_cast<bf16_t*>(smem);
  bf16_t* dOs = Qs + BLK * PR;
  bf16_t* Ks = dOs + BLK * PR;
  bf16_t* Vs = Ks + BLK * PR;
  bf16_t* Kt = Vs + BLK * PR;   // [128][PT]
  bf16_t* dSs = Kt + DH * PT;   // [64][PT] dS, high part
  bf16_t* dSl = dSs + BLK * PT; // low part
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const int64_t qs = (int64_t)a.heads * DH, ks = (int64_t)a.kv_heads * DH;
  load_block(Qs, nullptr, a.q + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
  load_block(dOs, nullptr, a.dout + ((int64_t)(E.row0 + q0) * a.heads + h) * DH, qs, nq, tid);
  float ls[4], dd[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qi = 16 * w + 4 * q4 + r;
    const int64_t t = (int64_t)h * a.N + E.row0 + q0 + qi;
    ls[r] = qi < nq ? a.lse[t] * kLog2e : INFINITY;
    dd[r] = qi < nq ? a.dsum[t] : 0.0f;
  }
  f32x4 dq[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) dq[j] = f32x4{0, 0, 0, 0};
  const float sl = a.scale * kLog2e;
  for (int kb = 0; kb <= qb; ++kb) {
    const int k0 = kb * BLK, nk = min(BLK, E.L - k0);
    __syncthreads();
    load_block(Ks, Kt, a.k + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
    load_block(Vs, nullptr, a.v + ((int64_t)(E.row0 + k0) * a.kv_heads + kh) * DH, ks, nk, tid);
    __syncthreads();
    f32x4 s[4], dp[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] = f32x4{0, 0, 0, 0}, dp[j] = f32x4{0, 0, 0, 0};
    mma_nt<DH / 32, 4>(Qs, PR, 16 * w, Ks, PR, 0, s, lane);
    mma_nt<DH / 32, 4>(dOs, PR, 16 * w, Vs, PR, 0, dp, lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kc = 16 * j + l16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qi = 16 * w + 4 * q4 + r;
        const bool ok = (k0 + kc <= q0 + qi) && (kc < nk);
        const float p = ok ? __builtin_amdgcn_exp2f(s[j][r] * sl - ls[r]) : 0.0f;
        const float ds = p * (dp[j][r] - dd[r]);
        const bf16_t hi = f2bf(ds);
        dSs[qi * PT + kc] = hi;
        dSl[qi * PT + kc] = f2bf(ds - bf2f(hi));
      }
    }
    __syncthreads();
    mma_nt<BLK / 32, 8>(dSs, PT, 16 * w, Kt, PT, 0, dq, lane);
    mma_nt<BLK / 32, 8>(dSl, PT, 16 * w, Kt, PT, 0, dq, lane);
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qi = 16 * w + 4 * q4 + r;
    if (qi >= nq) continue;
    bf16_t* dqr = a.dq + ((int64_t)(E.row0 + q0 + qi) * a.heads + h) * DH;
#pragma unroll
    for (int j = 0; j < 8; ++j) dqr[16 * j + l16] = f2bf(dq[j][r] * a.scale);
  }
}

size_t attn_lds_bytes(int kernel) {
  if (kernel == 0) return (size_t)(2 * BLK * PR + DH * PT + 2 * BLK * PT) * 2;
  if (kernel == 1) return (size_t)(4 * BLK * PR + 2 * DH * PT + 4 * BLK * PT) * 2 + 2 * BLK * 4;
  return (size_t)(4 * BLK * PR + DH * PT + 2 * BLK * PT) * 2;
}

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
  if (kernel == 0) hipLaunchKernelGGL(attn_fwd_stats_kernel, dim3(wgs), dim3(256), lds, s, a, b);
  if (kernel == 1) hipLaunchKernelGGL(attn_dkdv_kernel, dim3(wgs), dim3(256), lds, s, a, b);
  if (kernel == 2) hipLaunchKernelGGL(attn_dq_kernel, dim3(wgs), dim3(256), lds, s, a, b);
  return hipGetLastError();
}

}  // namespace attt
