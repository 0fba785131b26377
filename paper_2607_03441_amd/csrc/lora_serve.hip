// Serving side of the episode adapters on gfx950: concurrent episodes decode through the
// shared base model, each with its own LoRA adapter, and the adapter trained by an update is
// swapped into serving (Appendix A; adapter of Sec. 3.1, rank and alpha in Appendix C).
//
// lora_fwd_kernel: grouped multi-adapter forward. The base product x W0^T is a plain GEMM the
// caller has written into y; this adds y <- RN(y + scale (x A^T) B^T) for every (episode,
// projection), in one launch for all of them. A job is one x (an episode's rows) with up to
// four projections reading it (q, k, v of a layer): x is read once for all their ranks.
//   Phase 1: U = x A^T on v_mfma_f32_16x16x32_bf16, 16 rows per wave over the contraction
//     (64 rows per 4-wave workgroup), or, for at most 16 rows (decoding), an 8-wave workgroup
//     whose waves take an eighth of d_in each, their partial U summed in LDS in a fixed order. x rows and adapter rows are 16-byte loads in the MFMA's own k order, the next
//     128-wide step in flight.
//     scale U (float32) stays in LDS: nothing goes through HBM between the phases.
//   Phase 2: per projection, 256-column chunks of B [d_out, rank] staged transposed in LDS;
//     each thread adds the rank-long dot products for 8 consecutive columns of up to 8 rows
//     to y in float32 and rounds once to bf16 (16-byte loads and stores of y).
//   A row block's outputs may be split over `ncs` workgroups (each recomputing phase 1) so
//   that few rows still fill the chip; logical workgroups are mapped so that consecutive ones
//   (the splits of one row block) run on one XCD and share its L2.
// lora_swap_kernel: the swap. float32 adapter tensors -> their bf16 serving copies, rounded to
// nearest even, every tensor of an adapter in one launch.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

namespace {
constexpr uint32_t kOOBF = 0x7FFFFFF0u;  // offset past every descriptor's range: loads return 0
constexpr int kUP = 65;                  // LDS pitch (floats) of a row of U
constexpr int kBC = 256;                 // output columns per phase-2 chunk
constexpr int kBP = kBC + 8;             // LDS pitch (bf16) of a rank row of the transposed B chunk
constexpr int kBtBytes = 64 * kBP * 2;
// LDS scratch of a W-wave workgroup: the waves' partial U [W][16][kUP] floats, later the B chunk
template <int W>
constexpr int scratch_bytes() { return W * 16 * kUP * 4 > kBtBytes ? W * 16 * kUP * 4 : kBtBytes; }

template <class Batch>
__device__ __forceinline__ int job_of(const Batch& b, int li) {
  int j = 0;
  while (j + 1 < b.count && b.j[j + 1].b_begin <= li) ++j;
  return __builtin_amdgcn_readfirstlane(j);
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
}  // namespace

// W waves: 4 (up to 64 rows per workgroup, 16 per wave, or 16 rows with d_in split four ways)
// or 8 (decoding: 16 rows, d_in split eight ways, twice the loads in flight per workgroup).
template <int NU, int W>
__global__ __launch_bounds__(64 * W) void lora_fwd_kernel(LoraFwdBatch b, int grid) {
  constexpr int NT = 64 * W;
  // hardware places workgroup i on XCD i % 8: give each XCD a contiguous range of logical ids
  const int per = grid >> 3;
  const int li = (int)(blockIdx.x & 7u) * per + (int)(blockIdx.x >> 3);
  if (li >= b.total) return;
  const int ji = job_of(b, li);
  const LoraFwdJob& J = b.j[ji];
  const int local = li - J.b_begin;
  const int rb = local / J.ncs, cs = local - rb * J.ncs;
  const int row0 = rb * J.rb;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  __shared__ __align__(16) float Uf[64 * kUP];
  __shared__ __align__(16) uint8_t scr[scratch_bytes<W>()];
  float* Up = reinterpret_cast<float*>(scr);    // phase 1: [wave][16][kUP] partial U
  bf16_t* Bt = reinterpret_cast<bf16_t*>(scr);  // phase 2: [rank][kBP] transposed B chunk

  // ---- phase 1 ------------------------------------------------------------------------
  const int d_in = J.d_in, nu = J.nu;
  const int rg = J.kw > 1 ? 0 : w;  // this wave's 16 rows
  const int kp = J.kw > 1 ? w : 0;  // this wave's share of d_in
  const int r0w = row0 + 16 * rg;
  const int nrows = max(0, min(16, J.rows - r0w));
  const bf16_t* xs = static_cast<const bf16_t*>(J.x) + (int64_t)min(r0w, J.rows) * d_in;
  const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(xs, nrows * d_in * 2);
  __amdgpu_buffer_rsrc_t ra[NU];
#pragma unroll
  for (int t = 0; t < NU; ++t)
    ra[t] = buffer_rsrc(t < nu ? J.u[t].A : xs, t < nu ? J.u[t].valid * d_in * 2 : 0);
  const int ns = (d_in + 127) / 128;
  const int spw = (ns + J.kw - 1) / J.kw;
  const int s_begin = kp * spw, s_end = min(ns, s_begin + spw);
  f32x4 acc[NU];
#pragma unroll
  for (int t = 0; t < NU; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  // step s, MFMA q: lane (l16, g) holds row l16 (x) / rank l16 (A) at k = 128 s + 32 q + 8 g .. +7
  auto load = [&](int s, u32x4 (&xa)[4], u32x4 (&ao)[NU][4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = s * 128 + q * 32 + g * 8;
      const uint32_t off = k < d_in ? (uint32_t)(l16 * d_in + k) * 2u : kOOBF;
      xa[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0));
#pragma unroll
      for (int t = 0; t < NU; ++t)
        if (t < nu) ao[t][q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(ra[t], off, 0, 0));
    }
  };
  auto mma = [&](const u32x4 (&xa)[4], const u32x4 (&ao)[NU][4]) {
#pragma unroll
    for (int t = 0; t < NU; ++t) {
      if (t >= nu) break;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, xa[q]),
                                                         __builtin_bit_cast(bf16x8, ao[t][q]), acc[t], 0, 0, 0);
    }
  };
  {
    u32x4 x0[4], a0[NU][4], x1[4], a1[NU][4];
    if (s_begin < s_end) load(s_begin, x0, a0);
    for (int s = s_begin; s < s_end; s += 2) {
      if (s + 1 < s_end) load(s + 1, x1, a1);
      mma(x0, a0);
      if (s + 1 < s_end) {
        if (s + 2 < s_end) load(s + 2, x0, a0);
        mma(x1, a1);
      }
    }
  }
  // D of a 16x16 tile: lane l, register v -> row 4 (l / 16) + v, rank l % 16
#pragma unroll
  for (int t = 0; t < NU; ++t) {
    if (t >= nu) break;
#pragma unroll
    for (int v = 0; v < 4; ++v) Up[(w * 16 + 4 * g + v) * kUP + 16 * t + l16] = acc[t][v];
  }
  __syncthreads();
  for (int i = tid; i < J.rb * 64; i += NT) {
    const int row = i >> 6, c = i & 63, t = c >> 4;
    if (t >= nu) continue;
    float sc = J.u[0].scale;
#pragma unroll
    for (int k = 1; k < NU; ++k)
      if (t == k) sc = J.u[k].scale;
    float v = Up[row * kUP + c];  // kw == 1: wave row/16 wrote row row%16 of its block here
    for (int k = 1; k < J.kw; ++k) v += Up[(16 * k + row) * kUP + c];  // kw > 1: fixed order
    Uf[row * kUP + c] = sc * v;
  }
  __syncthreads();  // Up is dead from here on; its space holds the B chunks

  // ---- phase 2 ------------------------------------------------------------------------
  const int og = tid & 31, rs = tid >> 5;  // 8 columns og*8 .. +7 of rows rs, rs + 2W, ...
  const int nri = (J.rb + 2 * W - 1) / (2 * W);
#pragma unroll 1
  for (int p = 0; p < kLoraMaxTiles; ++p) {
    if (p >= J.no) break;
    const LoraFwdOut& O = J.o[p];
    const int d_out = O.d_out, rank = O.rank, u0 = O.u0;
    const int cw = (((d_out + J.ncs - 1) / J.ncs) + 7) & ~7;
    const int o_lo = cs * cw, o_hi = min(d_out, o_lo + cw);
    const bf16_t* B = static_cast<const bf16_t*>(O.B);
    bf16_t* y = static_cast<bf16_t*>(O.y);
    for (int oc = o_lo; oc < o_hi; oc += kBC) {
      const int nvo = min(kBC, o_hi - oc);  // a multiple of 8
      // B[oc .. oc + nvo)[0 .. rank) is contiguous: 16-byte loads, scattered into Bt[c][o]
      const int nel = nvo * rank;
      const bf16_t* src = B + (int64_t)oc * rank;
      for (int i8 = tid * 8; i8 < nel; i8 += NT * 8) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(src + i8);
        int o = i8 / rank, c = i8 - o * rank;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          Bt[c * kBP + o] = (bf16_t)((e & 1) ? (v[e >> 1] >> 16) : (v[e >> 1] & 0xFFFFu));
          if (++c == rank) c = 0, ++o;
        }
      }
      __syncthreads();
      const int ocol = og * 8;
      if (ocol < nvo) {
        // this thread's rows of y, loaded before the rank loop so that their latency overlaps it
        u32x4 yv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (i >= nri) break;
          const int rl = rs + 2 * W * i, row = row0 + rl;
          yv[i] = u32x4{0u, 0u, 0u, 0u};
          if (rl < J.rb && row < J.rows)
            yv[i] = *reinterpret_cast<const u32x4*>(y + (int64_t)row * d_out + oc + ocol);
        }
        float a[8][8];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int e = 0; e < 8; ++e) a[i][e] = 0.0f;
        for (int c = 0; c < rank; ++c) {
          const u32x4 bw = *reinterpret_cast<const u32x4*>(Bt + c * kBP + ocol);
          float bv[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) bv[2 * e] = bf_lo(bw[e]), bv[2 * e + 1] = bf_hi(bw[e]);
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            if (i >= nri) break;
            const float u = Uf[min(rs + 2 * W * i, 63) * kUP + u0 + c];
#pragma unroll
            for (int e = 0; e < 8; ++e) a[i][e] = fmaf(u, bv[e], a[i][e]);
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (i >= nri) break;
          const int rl = rs + 2 * W * i;
          const int row = row0 + rl;
          if (rl >= J.rb || row >= J.rows) continue;
          u32x4 out;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            out[e] = pack_bf16x2(bf_lo(yv[i][e]) + a[i][2 * e], bf_hi(yv[i][e]) + a[i][2 * e + 1]);
          *reinterpret_cast<u32x4*>(y + (int64_t)row * d_out + oc + ocol) = out;
        }
      }
      __syncthreads();  // Bt is rewritten by the next chunk
    }
  }
}

__global__ __launch_bounds__(256) void lora_swap_kernel(LoraSwapBatch b) {
  const int ji = job_of(b, (int)blockIdx.x);
  const LoraSwapJob J = b.j[ji];
  const int64_t i0 = ((int64_t)((int)blockIdx.x - J.b_begin) * 256 + threadIdx.x) * 8;
  if (i0 >= J.n) return;
  if (J.vec && i0 + 8 <= J.n) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(J.src + i0);
    const f32x4 c = *reinterpret_cast<const f32x4*>(J.src + i0 + 4);
    u32x4 o;
    o[0] = pack_bf16x2(a[0], a[1]);
    o[1] = pack_bf16x2(a[2], a[3]);
    o[2] = pack_bf16x2(c[0], c[1]);
    o[3] = pack_bf16x2(c[2], c[3]);
    *reinterpret_cast<u32x4*>(J.dst + i0) = o;
  } else {
    for (int64_t i = i0; i < J.n && i < i0 + 8; ++i) J.dst[i] = (uint16_t)f32_to_bf16_bits(J.src[i]);
  }
}

template <int W>
static void launch_fwd_w(int nu, const LoraFwdBatch& b, int grid, hipStream_t s) {
  switch (nu) {
    case 1: hipLaunchKernelGGL((lora_fwd_kernel<1, W>), dim3(grid), dim3(64 * W), 0, s, b, grid); break;
    case 2: hipLaunchKernelGGL((lora_fwd_kernel<2, W>), dim3(grid), dim3(64 * W), 0, s, b, grid); break;
    case 3: hipLaunchKernelGGL((lora_fwd_kernel<3, W>), dim3(grid), dim3(64 * W), 0, s, b, grid); break;
    default: hipLaunchKernelGGL((lora_fwd_kernel<4, W>), dim3(grid), dim3(64 * W), 0, s, b, grid); break;
  }
}

hipError_t launch_lora_fwd(int nu, int waves, const LoraFwdBatch& b, hipStream_t s) {
  if (b.total <= 0) return hipSuccess;
  const int grid = (b.total + 7) & ~7;
  KernelTimer t(K_LORA_FWD, s);
  if (waves == 8)
    launch_fwd_w<8>(nu, b, grid, s);
  else
    launch_fwd_w<4>(nu, b, grid, s);
  return hipGetLastError();
}

hipError_t launch_lora_swap(const LoraSwapBatch& b, int blocks, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_SWAP, s);
  hipLaunchKernelGGL(lora_swap_kernel, dim3(blocks), dim3(256), 0, s, b);
  return hipGetLastError();
}

}  // namespace attt
