// Token-weighted cross-entropy through a frozen LM head (Sec. 3.3, Eq. 10) on gfx950: the
// forward of both dtypes, the float32 backward, and the row and episode kernels around the bf16
// backward, whose two contractions run fused in one persistent kernel (ce_fused.hip).
//
// Forward (logits never leave the chip): one GEMM z = h W^T over (vocab tile, row tile) whose
// epilogue reduces every row of the tile to (max, sum exp(z - max)). A row kernel merges the
// partials into lse and w * CE; an episode kernel sums those in a fixed order into
// loss_e = (1/L_e) sum w_t CE_t.
//
// bf16 forward + backward: every row takes its own label logit r_t = z_{t,y_t} (ce_label_logit,
// one dot product per row) as the exponent reference, so the fused kernel forms
// e_tv = exp(z_tv - r_t) without knowing lse:
//     sigma_t = sum_{v != y_t} e_tv,   lse_t = r_t + log1p(sigma_t),   CE_t = log1p(sigma_t)
//     dL/dh_t = (w_t / L_e) (U_t - sigma_t W_{y_t}) / (1 + sigma_t),  U_t = sum_{v != y_t} e_tv W_v
// which is (w_t / L_e)(softmax(z_t) - onehot(y_t)) W rewritten; the label term is kept out of
// the sums, so nothing cancels when p_y is close to 1. ce_row_final turns the fused kernel's
// per-(row, vocab tile) sums into sigma, lse and the row losses. r_t is one of the row's logits,
// so sigma never underflows; a logit more than 64 above r_t (a label with probability below
// e^-64) could overflow e and raises a flag, on which the exact path (forward lse, then the fused
// kernel on coef exp(z - lse)) reruns in full, overwriting the outputs. Its kernels read the flag
// first and return at once when it is clear.
//
// bf16 GEMMs: MFMA v_mfma_f32_32x32x16_bf16 through the core in gemm_core.hpp (256x256 tiles on 8
// waves, 128x128 on 4 for small problems; XCD-aware tile order).
// f32 path: plain VALU tiles (64x64, 4x4 per thread) running the three-GEMM algorithm (forward,
// dZ = coef (softmax - onehot) staged per block of rows and vocabulary, dH = dZ W); it serves the
// float32 configuration.
#include "common.hpp"
#include "gemm_core.hpp"
#include "internal.hpp"

namespace attt {


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

// Rows [r0, r0 + R) after the fused backward: sigma_t = sum of the vocab-tile partials (fixed
// order), lse_t = r_t + log1p(sigma_t), row loss w_t log1p(sigma_t), and (when sa, sb are given)
// the row scales coef / (1 + sigma), coef sigma / (1 + sigma). One wave per row.
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
    if (sa) sa[row] = c * inv;
    if (sb) sb[row] = c * (sum * inv);
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
      // outside the contract: the row's loss term becomes NaN instead of reading stale memory
      if ((y < 0 || y >= V) && tn == 0 && tx == 0) label_logit[row] = __int_as_float(0x7FC00000);
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
    const bool bad = y < 0 || y >= V;  // outside the contract: NaN gradient row
    for (int j = 0; j < 4; ++j) {
      const int cl = n0 + tx * 4 + j, col = c0 + cl;
      float g = 0.0f;
      if (col < V) g = bad ? __int_as_float(0x7FC00000) : c * (expf(acc[i][j] - l) - (col == y ? 1.0f : 0.0f));
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

hipError_t launch_ce_row_final(int r0, int R, const float* sig_part, int n_vb, const float* label_logit,
                               const float* weights, const float* coef, float* lse, float* rowloss,
                               float* sa, float* sb, hipStream_t s) {
  if (R == 0) return hipSuccess;
  KernelTimer t(K_CE_ROW_REDUCE, s);
  hipLaunchKernelGGL(ce_row_final_kernel, dim3((R + 3) / 4), dim3(256), 0, s, r0, R, sig_part, n_vb,
                     label_logit, weights, coef, lse, rowloss, sa, sb);
  return hipGetLastError();
}

hipError_t launch_ce_bwd_dz(const float* h, const float* W, const int32_t* labels, const float* lse,
                            const float* coef, int r0, int R, int d, int c0, int Vc, int V, float* dz, int ldz,
                            hipStream_t s) {
  if (R == 0) return hipSuccess;
  const int tm = (R + kVT - 1) / kVT, tn = (Vc + kVT - 1) / kVT;
  const int cend = min(c0 + Vc, V);
  KernelTimer tt(K_CE_BWD_DZ, s);
  hipLaunchKernelGGL(ce_dz_f32_kernel, dim3(tm * tn), dim3(256), 0, s, h, W, labels, lse, coef, r0, R, d, c0, cend,
                     V, tm, dz, ldz);
  return hipGetLastError();
}

hipError_t launch_ce_bwd_dh(const float* dz, int ldz, const float* W, int r0, int R, int d, int c0, int K, int V,
                            float* grad, bool first, hipStream_t s) {
  if (R == 0) return hipSuccess;
  const int tm = (R + kVT - 1) / kVT, tn = (d + kVT - 1) / kVT;
  KernelTimer tt(K_CE_BWD_DH, s);
  hipLaunchKernelGGL(ce_dh_f32_kernel, dim3(tm * tn), dim3(256), 0, s, dz, ldz, W, r0, R, d, c0, K, V - c0, tm, grad,
                     first ? 1 : 0);
  return hipGetLastError();
}

}  // namespace attt
