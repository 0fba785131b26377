// LoRA adapter gradients (episode-specific adapter, Sec. 3.1; rank / alpha, Appendix C) on
// gfx950, for a group of adapted projections in one launch per pass.
//
// With U = x A^T and scale s:   dB = s dy^T U,   dA = (s dy B)^T x.
// Pass 1 (lora_u_kernel): per 128-row tile, sU^T = s (x A^T)^T and dU^T = s (dy B)^T,
//   contractions over d_in / d_out on MFMA 16x16x32 (rank padded to 16). Each lane streams
//   64 contiguous bytes of an x (dy) row per step; the four MFMAs of the step take the four
//   16-byte pieces, and the adapter operand in LDS is read with the same k order, so the
//   result is the same sum while the row reads stay fully coalesced. The two results are
//   stored transposed ([rank_pad, rows]) in the operand dtype for pass 2.
// Pass 2 (lora_dadb_kernel): dA^T-style products over the rows: out[c, k] = sum_t
//   dU^T[c, t] x[t, k] (and U^T dy for dB). The contraction runs over rows, which are the
//   slow index of x, so a 32-row x 64-column tile of x is written transposed into LDS
//   (16-bit stores) and read back as K-contiguous MFMA operands. Rows are split into
//   `splits` ranges whose float32 partials go to the workspace.
// Reduce (lora_reduce_kernel): sums the split partials in a fixed order and adds them to
//   dA [r, d_in] and dB [d_out, r]. No float atomics: results are bit-reproducible.
// The float32 path uses plain VALU loops with the same workspace layout.
#include "common.hpp"
#include "internal.hpp"

namespace attt {

template <class T>
__device__ __forceinline__ int find_job(const LoraBatch& b, int bid, T member) {
  int j = 0;
  while (j + 1 < b.count && b.j[j + 1].*member <= bid) ++j;
  return j;
}

constexpr int kP1KB = 128;  // pass-1 contraction block
constexpr int kP1Pitch = kP1KB + 8;

// ------------------------------------------------------------------------------------------
// bf16 pass 1
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_u_bf16_kernel(LoraBatch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x, &LoraJob::b1_begin);
  const LoraJob J = b.j[ji];
  const int local = (int)blockIdx.x - J.b1_begin;
  const int tiles = J.rows_pad / kLoraRowTile;
  const int kind = local / tiles;  // 0: U from (x, A); 1: dU from (dy, B)
  const int rt = local % tiles;
  const bf16_t* src = static_cast<const bf16_t*>(kind == 0 ? J.x : J.dy);
  const int kdim = kind == 0 ? J.d_in : J.d_out;
  const bf16_t* Al = static_cast<const bf16_t*>(J.A);  // [rank, d_in]
  const bf16_t* Bl = static_cast<const bf16_t*>(J.B);  // [d_out, rank]
  bf16_t* outT = reinterpret_cast<bf16_t*>(ws + (kind == 0 ? J.ut_off : J.dut_off));

  __shared__ __align__(16) bf16_t lop[64 * kP1Pitch];  // adapter operand [c][k] for this block
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int nct = J.rp / 16;
  f32x4 acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[a][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int row_base = rt * kLoraRowTile + wave * 32;

  for (int kb = 0; kb < kdim; kb += kP1KB) {
    __syncthreads();
    if (kind == 0) {
      for (int idx = tid; idx < J.rp * 16; idx += 256) {
        const int c = idx >> 4, ch = idx & 15;
        const int k = kb + ch * 8;
        u32x4 v = u32x4{0u, 0u, 0u, 0u};
        if (c < J.rank && k < kdim) v = *reinterpret_cast<const u32x4*>(Al + (int64_t)c * J.d_in + k);
        *reinterpret_cast<u32x4*>(lop + c * kP1Pitch + ch * 8) = v;
      }
    } else {
      for (int idx = tid; idx < J.rp * kP1KB; idx += 256) {
        const int k = idx / J.rp, c = idx % J.rp;
        bf16_t v = 0;
        if (c < J.rank && kb + k < kdim) v = Bl[(int64_t)(kb + k) * J.rank + c];
        lop[c * kP1Pitch + k] = v;
      }
    }
    __syncthreads();
    u32x4 xa[2][4];
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int row = row_base + a * 16 + l16;
      const bf16_t* p = src + (int64_t)row * kdim + kb + g * 32;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int k = kb + g * 32 + q * 8;
        xa[a][q] = (row < J.rows && k < kdim) ? *reinterpret_cast<const u32x4*>(p + q * 8)
                                              : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (c >= nct) break;
        const bf16x8 bv = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(lop + (c * 16 + l16) * kP1Pitch + g * 32 + q * 8));
#pragma unroll
        for (int a = 0; a < 2; ++a)
          acc[a][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, xa[a][q]),
                                                              bv, acc[a][c], 0, 0, 0);
      }
    }
  }
  // D[i][j] of a 16x16 tile: lane l, register v -> row 4*(l/16) + v, column l%16.
#pragma unroll
  for (int a = 0; a < 2; ++a) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c >= nct) break;
      const int col = c * 16 + l16;
      const int row0 = row_base + a * 16 + g * 4;
      uint2 pk;
      pk.x = pack_bf16x2(J.scale * acc[a][c][0], J.scale * acc[a][c][1]);
      pk.y = pack_bf16x2(J.scale * acc[a][c][2], J.scale * acc[a][c][3]);
      *reinterpret_cast<uint2*>(outT + (int64_t)col * J.rows_pad + row0) = pk;
    }
  }
}

// ------------------------------------------------------------------------------------------
// bf16 pass 2
// ------------------------------------------------------------------------------------------
constexpr int kP2Pitch = kLoraTStep + 8;  // LDS row pitch (bf16) of the transposed tile

__global__ __launch_bounds__(256) void lora_dadb_bf16_kernel(LoraBatch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x, &LoraJob::b2_begin);
  const LoraJob J = b.j[ji];
  int local = (int)blockIdx.x - J.b2_begin;
  const int cba = (J.d_in + kLoraColTile - 1) / kLoraColTile;
  const int cbb = (J.d_out + kLoraColTile - 1) / kLoraColTile;
  const int sp = local / (cba + cbb);
  local %= (cba + cbb);
  const int kind = local < cba ? 0 : 1;  // 0: dA from (dU^T, x); 1: dB from (sU^T, dy)
  const int cb = kind == 0 ? local : local - cba;
  const int cols = kind == 0 ? J.d_in : J.d_out;
  const bf16_t* src = static_cast<const bf16_t*>(kind == 0 ? J.x : J.dy);
  const bf16_t* lt = reinterpret_cast<const bf16_t*>(ws + (kind == 0 ? J.dut_off : J.ut_off));
  float* part = reinterpret_cast<float*>(ws + (kind == 0 ? J.pa_off : J.pb_off));
  const int col0 = cb * kLoraColTile;
  const int tper = ((J.rows_pad / J.splits + kLoraTStep - 1) / kLoraTStep) * kLoraTStep;
  const int t_begin = sp * tper;
  const int t_end = min(J.rows_pad, t_begin + tper);

  __shared__ __align__(16) bf16_t xs[kLoraColTile * kP2Pitch];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int nct = J.rp / 16;
  const int ld_t = tid >> 3, ld_c = (tid & 7) * 8;  // staging: row t, 8 columns
  f32x4 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int t0 = t_begin; t0 < t_end; t0 += kLoraTStep) {
    const int t = t0 + ld_t;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (t < J.rows && col0 + ld_c < cols)
      v = *reinterpret_cast<const u32x4*>(src + (int64_t)t * cols + col0 + ld_c);
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xs[(ld_c + 2 * e) * kP2Pitch + ld_t] = (bf16_t)(v[e] & 0xFFFFu);
      xs[(ld_c + 2 * e + 1) * kP2Pitch + ld_t] = (bf16_t)(v[e] >> 16);
    }
    __syncthreads();
    const bf16x8 bv = __builtin_bit_cast(
        bf16x8, *reinterpret_cast<const u32x4*>(xs + (wave * 16 + l16) * kP2Pitch + g * 8));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c >= nct) break;
      const bf16x8 av = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const u32x4*>(lt + (int64_t)(c * 16 + l16) * J.rows_pad + t0 + g * 8));
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[c], 0, 0, 0);
    }
  }
  const int col = col0 + wave * 16 + l16;
  if (col < cols) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c >= nct) break;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = c * 16 + g * 4 + v;
        part[((int64_t)sp * J.rp + r) * cols + col] = acc[c][v];
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// f32 passes (VALU)
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_u_f32_kernel(LoraBatch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x, &LoraJob::b1_begin);
  const LoraJob J = b.j[ji];
  const int local = (int)blockIdx.x - J.b1_begin;
  const int tiles = J.rows_pad / kLoraRowTile;
  const int kind = local / tiles, rt = local % tiles;
  const float* src = static_cast<const float*>(kind == 0 ? J.x : J.dy);
  const int kdim = kind == 0 ? J.d_in : J.d_out;
  const float* Al = static_cast<const float*>(J.A);
  const float* Bl = static_cast<const float*>(J.B);
  float* outT = reinterpret_cast<float*>(ws + (kind == 0 ? J.ut_off : J.dut_off));
  for (int idx = threadIdx.x; idx < kLoraRowTile * J.rp; idx += blockDim.x) {
    const int rl = idx % kLoraRowTile, c = idx / kLoraRowTile;
    const int row = rt * kLoraRowTile + rl;
    float s = 0.0f;
    if (row < J.rows && c < J.rank) {
      const float* xr = src + (int64_t)row * kdim;
      if (kind == 0)
        for (int k = 0; k < kdim; ++k) s = fmaf(xr[k], Al[(int64_t)c * J.d_in + k], s);
      else
        for (int k = 0; k < kdim; ++k) s = fmaf(xr[k], Bl[(int64_t)k * J.rank + c], s);
    }
    outT[(int64_t)c * J.rows_pad + row] = J.scale * s;
  }
}

__global__ __launch_bounds__(256) void lora_dadb_f32_kernel(LoraBatch b, uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x, &LoraJob::b2_begin);
  const LoraJob J = b.j[ji];
  int local = (int)blockIdx.x - J.b2_begin;
  const int cba = (J.d_in + kLoraColTile - 1) / kLoraColTile;
  const int cbb = (J.d_out + kLoraColTile - 1) / kLoraColTile;
  const int sp = local / (cba + cbb);
  local %= (cba + cbb);
  const int kind = local < cba ? 0 : 1;
  const int cb = kind == 0 ? local : local - cba;
  const int cols = kind == 0 ? J.d_in : J.d_out;
  const float* src = static_cast<const float*>(kind == 0 ? J.x : J.dy);
  const float* lt = reinterpret_cast<const float*>(ws + (kind == 0 ? J.dut_off : J.ut_off));
  float* part = reinterpret_cast<float*>(ws + (kind == 0 ? J.pa_off : J.pb_off));
  const int tper = ((J.rows_pad / J.splits + kLoraTStep - 1) / kLoraTStep) * kLoraTStep;
  const int t_begin = sp * tper;
  const int t_end = min(J.rows, t_begin + tper);
  const int col = cb * kLoraColTile + (threadIdx.x & 63);
  for (int c = threadIdx.x >> 6; c < J.rp; c += 4) {
    float s = 0.0f;
    if (col < cols)
      for (int t = t_begin; t < t_end; ++t)
        s = fmaf(lt[(int64_t)c * J.rows_pad + t], src[(int64_t)t * cols + col], s);
    if (col < cols) part[((int64_t)sp * J.rp + c) * cols + col] = s;
  }
}

// ------------------------------------------------------------------------------------------
// Ordered reduction of the split partials into dA, dB (+=).
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lora_reduce_kernel(LoraBatch b, const uint8_t* __restrict__ ws) {
  const int ji = find_job(b, (int)blockIdx.x, &LoraJob::b3_begin);
  const LoraJob J = b.j[ji];
  const int64_t idx = (int64_t)((int)blockIdx.x - J.b3_begin) * blockDim.x + threadIdx.x;
  const int64_t na = (int64_t)J.rank * J.d_in, nb = (int64_t)J.d_out * J.rank;
  if (idx < na) {
    const int c = (int)(idx / J.d_in), k = (int)(idx % J.d_in);
    const float* p = reinterpret_cast<const float*>(ws + J.pa_off);
    float s = 0.0f;
    for (int sp = 0; sp < J.splits; ++sp) s += p[((int64_t)sp * J.rp + c) * J.d_in + k];
    J.dA[idx] += s;
  } else if (idx < na + nb) {
    const int64_t i2 = idx - na;
    const int o = (int)(i2 / J.rank), c = (int)(i2 % J.rank);
    const float* p = reinterpret_cast<const float*>(ws + J.pb_off);
    float s = 0.0f;
    for (int sp = 0; sp < J.splits; ++sp) s += p[((int64_t)sp * J.rp + c) * J.d_out + o];
    J.dB[i2] += s;
  }
}

// ------------------------------------------------------------------------------------------
hipError_t launch_lora_pass1(int dtype, const LoraBatch& b, int blocks, uint8_t* ws, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_U, s);
  if (dtype == 1)
    hipLaunchKernelGGL(lora_u_bf16_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  else
    hipLaunchKernelGGL(lora_u_f32_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  return hipGetLastError();
}

hipError_t launch_lora_pass2(int dtype, const LoraBatch& b, int blocks, uint8_t* ws, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_DADB, s);
  if (dtype == 1)
    hipLaunchKernelGGL(lora_dadb_bf16_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  else
    hipLaunchKernelGGL(lora_dadb_f32_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  return hipGetLastError();
}

hipError_t launch_lora_reduce(const LoraBatch& b, int blocks, uint8_t* ws, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  KernelTimer t(K_LORA_REDUCE, s);
  hipLaunchKernelGGL(lora_reduce_kernel, dim3(blocks), dim3(256), 0, s, b, ws);
  return hipGetLastError();
}

}  // namespace attt
