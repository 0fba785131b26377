// LoRA adapter gradients (episode-specific adapter, Sec. 3.1; rank / alpha, Appendix C) on
// gfx950, for a group of adapted projections.
//
// With U = x A^T and scale s:   dB = s dy^T U,   dA = (s dy B)^T x.
// Work is cut into rank tiles of 16 (rank padded to 16). Projections that read the same
// input x (q, k, v of one layer) form one job of up to four tiles, so x is streamed once per
// pass for all of them; dy differs per projection.
//   B^T (lora_bt_kernel): B [d_out, r] -> B^T [r_pad, d_out] (zero rows past r), so both
//     adapter operands are row-major [rank, k].
//   Pass 1 (lora_p1_*): per 64 rows of x (or dy), s U^T = s (x A^T)^T (or s (dy B)^T) for all
//     tiles of the job, on MFMA 16x16x32; each of the workgroup's four waves owns 16 rows over
//     the whole contraction. Rows are 16-byte loads in the MFMA's own k order (each instruction
//     covers 64 contiguous bytes of 16 rows), two steps in flight; the adapter operand slice of
//     each step is staged once per workgroup in LDS and shared by its waves. Results are
//     stored transposed, per tile as two bf16 planes hi = RN(v), lo = RN(v - hi) of the float32
//     value v ([2][16, rows_pad]), so pass 2 contracts with ~16 significant bits.
//   Pass 2 (lora_p2_*): out[c, k] = sum_t L[c, t] src[t, k] with (L, src) = (s dU^T, x) for dA
//     and (s U^T, dy) for dB. The contraction runs over rows, the slow index of src, so 64-row
//     x 64-column tiles of src are written transposed into LDS (two rows per 32-bit store,
//     double-buffered, one barrier per step) and read back as K-contiguous MFMA operands; the
//     step's slice of L (both planes) is staged in LDS once per workgroup beside them.
//     Rows are split into `splits` ranges whose float32 partials go to the workspace.
//   Reduce (lora_reduce_kernel): sums the split partials in a fixed order and adds them to
//     dA [r, d_in] and dB [d_out, r]. No float atomics: results are bit-reproducible.
// The float32 path runs the same jobs with plain VALU loops.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

// Job of workgroup `bid`; wave-uniform (made explicit so the descriptors built from the job's
// pointers live in scalar registers).
template <class Batch>
__device__ __forceinline__ int find_job(const Batch& b, int bid) {
  int j = 0;
  while (j + 1 < b.count && b.j[j + 1].b_begin <= bid) ++j;
  return __builtin_amdgcn_readfirstlane(j);
}

// ------------------------------------------------------------------------------------------
// B [d_out, rank] -> B^T [rp, d_out], zero rows rank .. rp-1 (bf16 or float, by element size).
// ------------------------------------------------------------------------------------------
template <class T>
__global__ __launch_bounds__(256) void lora_bt_kernel(LoraBTBatch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraBTJob J = b.j[ji];
  const int64_t idx = (int64_t)((int)blockIdx.x - J.b_begin) * 256 + threadIdx.x;
  if (idx >= (int64_t)J.rp * J.d_out) return;
  const int c = (int)(idx / J.d_out), k = (int)(idx % J.d_out);
  const T* B = static_cast<const T*>(J.B);
  T v = T(0);
  if (c < J.rank) v = B[(int64_t)k * J.rank + c];
  reinterpret_cast<T*>(ws + J.bt_off)[idx] = v;
}

// ------------------------------------------------------------------------------------------
// bf16 pass 1
// ------------------------------------------------------------------------------------------
constexpr uint32_t kOOB = 0x7FFFFFF0u;  // offset past every descriptor's range: loads return 0

// A workgroup takes kLoraP1Rows = 64 rows, each of its four waves 16 of them over the whole
// contraction. The rank tiles' operand slices of every 128-wide step ([16, 128] per tile) are
// loaded once per workgroup into LDS (double-buffered, rows padded to kP1Pitch elements so the
// sixteen rows one fragment read touches fall in distinct banks) and shared by the four waves,
// so the operand traffic from L2 is a quarter of what per-wave fragment loads would cost. The
// rows of step s+2 are in flight while step s runs. NT is the largest tile count of the batch;
// a job with fewer tiles skips the rest.
constexpr int kP1Pitch = kLoraKBlock + 8;
static_assert(kLoraP1Rows == 64, "four waves of 16 rows");

template <int NT>
__global__ __launch_bounds__(256) void lora_p1_bf16_kernel(LoraP1Batch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraP1Job& Jr = b.j[ji];
  const int rt = (int)blockIdx.x - Jr.b_begin;
  const int kdim = Jr.kdim, nt = Jr.nt;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  // this wave's 16 rows; rows past the input read as zero through the descriptor range
  const int row0 = rt * kLoraP1Rows + wave * 16;
  const int nrows = max(0, min(16, Jr.rows - row0));
  const bf16_t* src = static_cast<const bf16_t*>(Jr.src) + (int64_t)min(row0, Jr.rows) * kdim;
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(src, nrows * kdim * 2);
  __amdgpu_buffer_rsrc_t ro[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
    ro[t] = buffer_rsrc(t < nt ? Jr.t[t].op : src, t < nt ? Jr.t[t].valid * kdim * 2 : 0);
  __shared__ __align__(16) bf16_t opl[2][NT][16 * kP1Pitch];
  const int ns = (kdim + kLoraKBlock - 1) / kLoraKBlock;

  // operand staging: thread -> operand row sr, 16-byte chunk sc of the step's 128 columns
  const int sr = tid >> 4, sc = tid & 15;
  u32x4 stg[NT];
  auto stage_load = [&](int s) {
    const int k = s * kLoraKBlock + sc * 8;
#pragma unroll
    for (int t = 0; t < NT; ++t)
      if (t < nt)
        stg[t] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(ro[t], k < kdim ? (uint32_t)(sr * kdim + k) * 2u : kOOB, 0, 0));
  };
  auto stage_store = [&](int buf) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
      if (t < nt) *reinterpret_cast<u32x4*>(&opl[buf][t][sr * kP1Pitch + sc * 8]) = stg[t];
  };
  // Step s of the rows: for MFMA q, lane (l16, g) holds row l16 at k = 128 s + 32 q + 8 g .. +7
  // (the MFMA's own k order; one load instruction covers 64 contiguous bytes of 16 rows); k at
  // or past kdim reads as zero.
  auto xload = [&](int s, u32x4 (&xa)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int k = s * kLoraKBlock + q * 32 + g * 8;
      xa[q] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, k < kdim ? (uint32_t)(l16 * kdim + k) * 2u : kOOB, 0, 0));
    }
  };
  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](int buf, const u32x4 (&xa)[4]) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t >= nt) break;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const u32x4 o = *reinterpret_cast<const u32x4*>(&opl[buf][t][l16 * kP1Pitch + q * 32 + g * 8]);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, xa[q]),
                                                         __builtin_bit_cast(bf16x8, o), acc[t], 0, 0, 0);
      }
    }
  };
  u32x4 x0[4], x1[4];
  stage_load(0);
  xload(0, x0);
  if (ns > 1) xload(1, x1);
  stage_store(0);
  __syncthreads();
  // Step s: the operand stage of s+1 in flight, the MFMAs of step s (LDS buffer s&1, rows
  // loaded two steps earlier), the rows of step s+2 into the registers just consumed, then
  // the stage of s+1 into the other buffer and one barrier. That buffer was last read in step
  // s-1, before the previous barrier.
  auto step = [&](int s, u32x4 (&xa)[4]) {
    if (s + 1 < ns) stage_load(s + 1);
    mma(s & 1, xa);
    if (s + 2 < ns) xload(s + 2, xa);
    if (s + 1 < ns) stage_store((s + 1) & 1);
    __syncthreads();
  };
  for (int s = 0; s < ns; s += 2) {
    step(s, x0);
    if (s + 1 < ns) step(s + 1, x1);
  }
  // D of a 16x16 tile: lane l, register v -> row 4*(l/16) + v, column l%16. The float32 result
  // v goes out as two bf16 planes, hi = RN(v) and lo = RN(v - hi) (v - hi is exact in float32),
  // so pass 2 contracts with hi + lo, about 16 significant bits instead of bf16's 8.
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t >= nt) break;
    bf16_t* outT = reinterpret_cast<bf16_t*>(ws + Jr.t[t].out_off);
    const float scale = Jr.t[t].scale;
    const int r = row0 + g * 4;
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = scale * acc[t][e];
    uint2 hi, lo;
    hi.x = pack_bf16x2(v[0], v[1]);
    hi.y = pack_bf16x2(v[2], v[3]);
    lo.x = pack_bf16x2(v[0] - bf16_bits_to_f32(hi.x & 0xFFFFu), v[1] - bf16_bits_to_f32(hi.x >> 16));
    lo.y = pack_bf16x2(v[2] - bf16_bits_to_f32(hi.y & 0xFFFFu), v[3] - bf16_bits_to_f32(hi.y >> 16));
    *reinterpret_cast<uint2*>(outT + (int64_t)l16 * Jr.rows_pad + r) = hi;
    *reinterpret_cast<uint2*>(outT + (int64_t)(16 + l16) * Jr.rows_pad + r) = lo;
  }
}

// ------------------------------------------------------------------------------------------
// bf16 pass 2
// ------------------------------------------------------------------------------------------
constexpr int kP2Pitch = kLoraTStep + 8;  // LDS row pitch (bf16) of the transposed tile

size_t lora_p2_lds(int max_nt) { return (size_t)(2 * kLoraColTile + 2 * max_nt * 32) * kP2Pitch * 2; }

__global__ __launch_bounds__(256) void lora_p2_bf16_kernel(LoraP2Batch b, int max_nt, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraP2Job& Jr = b.j[ji];
  const int cols = Jr.cols, nt = Jr.nt;
  const int ncb = (cols + kLoraColTile - 1) / kLoraColTile;
  const int local = (int)blockIdx.x - Jr.b_begin;
  const int sp = local / ncb, cb = local % ncb;
  const int col0 = cb * kLoraColTile;
  const int tper = ((Jr.rows_pad / Jr.splits + kLoraTStep - 1) / kLoraTStep) * kLoraTStep;
  const int t_begin = sp * tper;
  const int t_end = min(Jr.rows_pad, t_begin + tper);

  // Dynamic LDS: xs[2][kLoraColTile * kP2Pitch], then lt[2][max_nt][32 * kP2Pitch], the step's
  // slice of every tile's L (planes hi, lo: 32 rows of kLoraTStep), shared by the workgroup's
  // four waves, which all contract with the same fragments. max_nt: the batch's largest nt.
  extern __shared__ __align__(16) uint8_t p2_smem[];
  bf16_t (*xs)[kLoraColTile * kP2Pitch] = reinterpret_cast<bf16_t (*)[kLoraColTile * kP2Pitch]>(p2_smem);
  bf16_t* lt_base = reinterpret_cast<bf16_t*>(p2_smem) + 2 * kLoraColTile * kP2Pitch;
  auto lt = [&](int buf, int t) { return lt_base + (buf * max_nt + t) * (32 * kP2Pitch); };
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  // staging: rows 2*pr, 2*pr+1 of the step, columns 8*cg .. 8*cg+7 of the tile
  const int pr = tid >> 3, cg = tid & 7;
  const bool cin = col0 + cg * 8 < cols;  // cols % 8 == 0: a column chunk is whole or absent
  // L staging: plane row lr (hi rows 0-15, lo rows 16-31), 8 consecutive t from 8*lk
  const int lr = tid >> 3, lk = tid & 7;
  const bf16_t* src = static_cast<const bf16_t*>(Jr.src);
  // a tile's pass-1 result: planes hi and lo, [2][16][rows_pad] bf16
  __amdgpu_buffer_rsrc_t rl[kLoraMaxTiles];
#pragma unroll
  for (int t = 0; t < kLoraMaxTiles; ++t)
    rl[t] = buffer_rsrc(ws + (t < nt ? Jr.t[t].lt_off : 0), t < nt ? 2 * 16 * Jr.rows_pad * 2 : 0);

  f32x4 acc[kLoraMaxTiles];
#pragma unroll
  for (int t = 0; t < kLoraMaxTiles; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Rows of step t0 go through a descriptor based at row t0 (offsets stay small) whose range
  // ends at the input's last row.
  auto load = [&](int t0, u32x4 (&v)[2], u32x4 (&la)[kLoraMaxTiles]) {
    const int nr = max(0, min(kLoraTStep, Jr.rows - t0));
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(src + (int64_t)t0 * cols, nr * cols * 2);
#pragma unroll
    for (int e = 0; e < 2; ++e)
      v[e] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, cin ? (uint32_t)((2 * pr + e) * cols + col0 + cg * 8) * 2u : kOOB, 0, 0));
#pragma unroll
    for (int t = 0; t < kLoraMaxTiles; ++t)
      if (t < nt)  // uniform: a job's tile count; unused tiles issue no load
        la[t] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rl[t], (uint32_t)(lr * Jr.rows_pad + t0 + lk * 8) * 2u, 0, 0));
  };
  u32x4 v0[2], v1[2], la0[kLoraMaxTiles], la1[kLoraMaxTiles];
  // One step: store its rows transposed (row pairs as 32-bit words) into buffer `buf` and the L
  // slices into lt[buf], one barrier, two MFMA k-steps of 32 rows, each as the hi and then the
  // lo plane of L. Both buffers `buf` were last read two steps earlier, before the previous
  // step's barrier.
  auto step = [&](int buf, const u32x4 (&v)[2], const u32x4 (&la)[kLoraMaxTiles]) {
    uint32_t* dst = reinterpret_cast<uint32_t*>(xs[buf]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo0 = v[0][e] & 0xFFFFu, hi0 = v[0][e] >> 16;
      const uint32_t lo1 = v[1][e] & 0xFFFFu, hi1 = v[1][e] >> 16;
      dst[((cg * 8 + 2 * e) * kP2Pitch + 2 * pr) >> 1] = lo0 | (lo1 << 16);
      dst[((cg * 8 + 2 * e + 1) * kP2Pitch + 2 * pr) >> 1] = hi0 | (hi1 << 16);
    }
#pragma unroll
    for (int t = 0; t < kLoraMaxTiles; ++t)
      if (t < nt) *reinterpret_cast<u32x4*>(lt(buf, t) + lr * kP2Pitch + lk * 8) = la[t];
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const bf16x8 bv = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(xs[buf] + (wave * 16 + l16) * kP2Pitch + ks * 32 + g * 8));
#pragma unroll
      for (int t = 0; t < kLoraMaxTiles; ++t) {
        if (t >= nt) break;
#pragma unroll
        for (int hl = 0; hl < 2; ++hl) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(lt(buf, t) + (hl * 16 + l16) * kP2Pitch + ks * 32 + g * 8);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), bv, acc[t], 0, 0, 0);
        }
      }
    }
  };
  if (t_begin < t_end) load(t_begin, v0, la0);
  for (int t0 = t_begin; t0 < t_end; t0 += 2 * kLoraTStep) {
    const bool two = t0 + kLoraTStep < t_end;
    if (two) load(t0 + kLoraTStep, v1, la1);
    step(0, v0, la0);
    if (!two) break;
    if (t0 + 2 * kLoraTStep < t_end) load(t0 + 2 * kLoraTStep, v0, la0);
    step(1, v1, la1);
  }
  const int col = col0 + wave * 16 + l16;
  if (col < cols) {
#pragma unroll
    for (int t = 0; t < kLoraMaxTiles; ++t) {
      if (t >= nt) break;
      float* part = reinterpret_cast<float*>(ws + Jr.t[t].part_off) + (int64_t)sp * 16 * cols;
#pragma unroll
      for (int v = 0; v < 4; ++v) part[(int64_t)(g * 4 + v) * cols + col] = acc[t][v];
    }
  }
}

// ------------------------------------------------------------------------------------------
// f32 passes (VALU), same jobs and workspace layout
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_p1_f32_kernel(LoraP1Batch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraP1Job& J = b.j[ji];
  const int rt = (int)blockIdx.x - J.b_begin;
  const float* src = static_cast<const float*>(J.src);
  for (int idx = threadIdx.x; idx < kLoraP1Rows * 16 * J.nt; idx += blockDim.x) {
    const int rl = idx % kLoraP1Rows, c = idx / kLoraP1Rows;  // c: rank within the job
    const int t = c >> 4, cr = c & 15;
    const int row = rt * kLoraP1Rows + rl;
    float s = 0.0f;
    if (row < J.rows && cr < J.t[t].valid) {
      const float* xr = src + (int64_t)row * J.kdim;
      const float* op = static_cast<const float*>(J.t[t].op) + (int64_t)cr * J.kdim;
      for (int k = 0; k < J.kdim; ++k) s = fmaf(xr[k], op[k], s);
    }
    reinterpret_cast<float*>(ws + J.t[t].out_off)[(int64_t)cr * J.rows_pad + row] = J.t[t].scale * s;
  }
}

__global__ __launch_bounds__(256) void lora_p2_f32_kernel(LoraP2Batch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraP2Job& J = b.j[ji];
  const int ncb = (J.cols + kLoraColTile - 1) / kLoraColTile;
  const int local = (int)blockIdx.x - J.b_begin;
  const int sp = local / ncb, cb = local % ncb;
  const int tper = ((J.rows_pad / J.splits + kLoraTStep - 1) / kLoraTStep) * kLoraTStep;
  const int t_begin = sp * tper;
  const int t_end = min(J.rows, t_begin + tper);
  const int col = cb * kLoraColTile + (threadIdx.x & 63);
  const float* src = static_cast<const float*>(J.src);
  for (int c = threadIdx.x >> 6; c < 16 * J.nt; c += 4) {
    const int t = c >> 4, cr = c & 15;
    const float* lt = reinterpret_cast<const float*>(ws + J.t[t].lt_off) + (int64_t)cr * J.rows_pad;
    float s = 0.0f;
    if (col < J.cols)
      for (int r = t_begin; r < t_end; ++r) s = fmaf(lt[r], src[(int64_t)r * J.cols + col], s);
    if (col < J.cols)
      reinterpret_cast<float*>(ws + J.t[t].part_off)[((int64_t)sp * 16 + cr) * J.cols + col] = s;
  }
}

// ------------------------------------------------------------------------------------------
// Ordered reduction of the split partials into dA, dB (+=). Partials of rank c of a problem
// live in its tile c/16: [tile][split][16][cols]. The split loop is unrolled so its loads are
// in flight together; the additions keep their order.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_reduce_kernel(LoraRedBatch b, const uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraRedJob J = b.j[ji];
  const int64_t idx = (int64_t)((int)blockIdx.x - J.b_begin) * blockDim.x + threadIdx.x;
  const int64_t na = (int64_t)J.rank * J.d_in, nb = (int64_t)J.d_out * J.rank;
  if (idx < na) {
    const int c = (int)(idx / J.d_in), k = (int)(idx % J.d_in);
    const float* p = reinterpret_cast<const float*>(ws + J.pa_off) +
                     ((int64_t)(c >> 4) * J.sa * 16 + (c & 15)) * J.d_in + k;
    float s = 0.0f;
#pragma unroll 8
    for (int sp = 0; sp < J.sa; ++sp) s += p[(int64_t)sp * 16 * J.d_in];
    J.dA[idx] += s;
  } else if (idx < na + nb) {
    const int64_t i2 = idx - na;
    const int o = (int)(i2 / J.rank), c = (int)(i2 % J.rank);
    const float* p = reinterpret_cast<const float*>(ws + J.pb_off) +
                     ((int64_t)(c >> 4) * J.sb * 16 + (c & 15)) * J.d_out + o;
    float s = 0.0f;
#pragma unroll 8
    for (int sp = 0; sp < J.sb; ++sp) s += p[(int64_t)sp * 16 * J.d_out];
    J.dB[i2] += s;
  }
}

// ------------------------------------------------------------------------------------------
// Adapter step of Eq. 2: p <- p - lr g in float32, the product and the difference each rounded
// to nearest (explicit roundings, no contraction into a fused multiply-add), then the bf16
// copy (round to nearest even) and the gradient reset when asked. 1024 elements per workgroup.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_sgd_kernel(LoraSgdBatch b, float lr, int zero_grad) {
  const int ji = find_job(b, (int)blockIdx.x);
  const LoraSgdJob J = b.j[ji];
  const int64_t base = (int64_t)((int)blockIdx.x - J.b_begin) * kLoraSgdPerBlock;
#pragma unroll
  for (int u = 0; u < kLoraSgdPerBlock / 256; ++u) {
    const int64_t i = base + u * 256 + threadIdx.x;
    if (i < J.n) {
#pragma clang fp contract(off)  // the product keeps its own rounding: no fused multiply-add
      const float t = lr * J.grad[i];
      const float p = J.param[i] - t;
      J.param[i] = p;
      if (J.param_bf16) J.param_bf16[i] = (uint16_t)f32_to_bf16_bits(p);
      if (zero_grad) J.grad[i] = 0.0f;
    }
  }
}

hipError_t launch_lora_sgd(const LoraSgdBatch& b, int blocks, float lr, int zero_grad, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_SGD, s);
  hipLaunchKernelGGL(lora_sgd_kernel, dim3(blocks), dim3(256), 0, s, b, lr, zero_grad);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------
hipError_t launch_lora_bt(int dtype, const LoraBTBatch& b, int blocks, uint8_t* ws, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_U, s);
  if (dtype == 1)
    hipLaunchKernelGGL(lora_bt_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, b, ws);
  else
    hipLaunchKernelGGL(lora_bt_kernel<float>, dim3(blocks), dim3(256), 0, s, b, ws);
  return hipGetLastError();
}

hipError_t launch_lora_pass1(int dtype, int nt, const LoraP1Batch& b, int blocks, uint8_t* ws,
                             hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_U, s);
  if (dtype != 1) {
    hipLaunchKernelGGL(lora_p1_f32_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  } else {
    switch (nt) {
      case 1: hipLaunchKernelGGL(lora_p1_bf16_kernel<1>, dim3(blocks), dim3(256), 0, s, b, ws); break;
      case 2: hipLaunchKernelGGL(lora_p1_bf16_kernel<2>, dim3(blocks), dim3(256), 0, s, b, ws); break;
      case 3: hipLaunchKernelGGL(lora_p1_bf16_kernel<3>, dim3(blocks), dim3(256), 0, s, b, ws); break;
      default: hipLaunchKernelGGL(lora_p1_bf16_kernel<4>, dim3(blocks), dim3(256), 0, s, b, ws); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_lora_pass2(int dtype, const LoraP2Batch& b, int blocks, uint8_t* ws, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_DADB, s);
  int max_nt = 1;
  for (int i = 0; i < b.count; ++i) max_nt = max(max_nt, b.j[i].nt);
  if (dtype == 1)
    hipLaunchKernelGGL(lora_p2_bf16_kernel, dim3(blocks), dim3(256), lora_p2_lds(max_nt), s, b, max_nt, ws);
  else
    hipLaunchKernelGGL(lora_p2_f32_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  return hipGetLastError();
}

hipError_t launch_lora_reduce(const LoraRedBatch& b, int blocks, uint8_t* ws, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_REDUCE, s);
  hipLaunchKernelGGL(lora_reduce_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  return hipGetLastError();
}

}  // namespace attt
