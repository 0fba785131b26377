// Host-side interfaces between the C ABI layer (api.cpp) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace attt {

// ---- kernel timing ---------------------------------------------------------------------
enum KernelId {
  K_NGRAM_COUNT = 0,
  K_NGRAM_WEIGHT,
  K_CE_FWD,
  K_CE_LABEL,
  K_CE_ROW_REDUCE,
  K_CE_LOSS,
  K_CE_HEAD_T,
  K_CE_BWD_DZ,
  K_CE_BWD_DH,
  K_CE_LOGIT_EXP,
  K_CE_GUARD,
  K_LORA_U,
  K_LORA_DADB,
  K_LORA_REDUCE,
  K_NUM_KERNELS
};

const char* kernel_name(int id);
bool timing_on();
void timing_record(int id, hipEvent_t start, hipEvent_t stop);

// Brackets one launch with events on its stream when timing is enabled.
struct KernelTimer {
  int id;
  hipStream_t stream;
  hipEvent_t a = nullptr, b = nullptr;
  KernelTimer(int id_, hipStream_t s) : id(id_), stream(s) {
    if (timing_on() && hipEventCreate(&a) == hipSuccess && hipEventCreate(&b) == hipSuccess)
      (void)hipEventRecord(a, stream);
    else
      a = b = nullptr;
  }
  ~KernelTimer() {
    if (a && b) {
      (void)hipEventRecord(b, stream);
      timing_record(id, a, b);
    }
  }
};

// ---- n-gram ----------------------------------------------------------------------------
constexpr int kQMax = 4096;        // query n-gram starts per partition (12-bit positions)
constexpr int kMaxN = 16;          // largest n
constexpr int kPartBatch = 32;     // partitions per launch (kernel-argument descriptors)
constexpr int kEpBatch = 64;       // episodes per launch

struct NgramPart {
  int64_t tok_base;            // first update token of the episode in `tokens`
  int64_t hist_base;           // first history token of the episode in `history`
  int64_t chunk_begin_global;  // first row of this partition in the partial-count array
  int32_t hist_ngrams;         // history n-gram starts of the episode: max(0, H_e - n + 1)
  int32_t q0;                  // first query start of this partition, relative to the episode
  int32_t qn;                  // query starts in this partition, 1 .. kQMax
  int32_t slots;               // LDS table size, power of two >= 2 * qn
  int32_t chunk_begin;         // first count-kernel block of this partition within the launch
  int32_t chunks;              // history chunks (count-kernel blocks) of the partition
};

struct NgramPartBatch {
  int32_t count;
  int32_t pad;
  NgramPart p[kPartBatch];
};

struct NgramEp {
  int64_t tok_base;
  int64_t chunk_base;  // partial-count row of the episode's first partition, first chunk
  int32_t L;
  int32_t chunks;      // chunks per partition (the same for every partition of the episode)
  int32_t block_begin;
  int32_t pad;
};

struct NgramEpBatch {
  int32_t count;
  int32_t pad;
  NgramEp e[kEpBatch];
};

size_t ngram_count_lds(int slots, int n);
hipError_t launch_ngram_count(const NgramPartBatch& b, int total_blocks, int max_slots,
                              const int32_t* history, const int32_t* tokens, int n,
                              uint16_t* partial, hipStream_t s);
hipError_t launch_ngram_weight(const NgramEpBatch& b, int total_blocks, int n, float w_min,
                               const uint16_t* partial, uint32_t* exposure, float* weights,
                               hipStream_t s);

// ---- weighted cross-entropy ------------------------------------------------------------
struct CeEp {
  int64_t row0;       // first row of the episode
  int32_t L;          // rows of the episode
  int32_t block_begin;
};

struct CeEpBatch {
  int32_t count;
  int32_t first;  // index of e[0] among all episodes of the call
  CeEp e[kEpBatch];
};

// Tile shapes of the LM-head GEMMs (bf16 MFMA path: 256x256 or 128x128; f32 path: 64x64).
struct CeGemmShape {
  int bm, bn;
};

// Forward: per (row, vocab tile) partial (max, sum exp); the f32 kernel also writes the label
// logits. `gate` (nullable): when non-null the kernels return at once unless *gate != 0.
hipError_t launch_ce_fwd(int dtype, CeGemmShape t, const void* h, const void* W,
                         const int32_t* labels, int N, int d, int V, float2* partials, int n_vb,
                         float* label_logit, const int* gate, hipStream_t s);
// bf16 label logits z_{t, y_t}; NaN for a label outside [0, V). Clears *flag when non-null.
hipError_t launch_ce_label(const void* h, const void* W, const int32_t* labels, int N, int d, int V,
                           float* label_logit, int* flag, hipStream_t s);
hipError_t launch_ce_row_reduce(const CeEpBatch& b, int total_blocks, const float2* partials,
                                int n_vb, const float* label_logit, const float* weights,
                                float* lse, float* coef, float* rowloss, const int* gate,
                                hipStream_t s);
hipError_t launch_ce_loss(const CeEpBatch& b, const float* rowloss, float* loss, const int* gate,
                          hipStream_t s);
// coef_t = w_t / L_e (256 rows per block).
hipError_t launch_ce_coef(const CeEpBatch& b, int total_blocks, const float* weights, float* coef,
                          hipStream_t s);
// W [V, d] -> WT [d, Vp] (bf16 only), zero columns V .. Vp-1.
hipError_t launch_ce_head_transpose(const void* W, int V, int d, int Vp, void* WT, hipStream_t s);
// bf16, label-referenced: e = exp(z - z_y) (0 at the label and past V) for rows [r0, r0+R) x
// vocab [c0, c0+Vc) into staging [R, ldz]; per (row, vocab tile of t.bm) sums into
// sig_part [N, n_vb]; sets *flag when a logit exceeds its reference by more than 64.
hipError_t launch_ce_logit_exp(CeGemmShape t, const void* h, const void* W, const int32_t* labels,
                               const float* label_logit, int r0, int R, int d, int c0, int Vc, int V,
                               float* sig_part, int n_vb, void* ez, int ldz, int* flag, hipStream_t s);
// Rows [r0, r0+R): sigma, lse, row loss and the dH row scales (sa, sb).
hipError_t launch_ce_row_final(int r0, int R, const float* sig_part, int n_vb, const float* label_logit,
                               const float* weights, const float* coef, float* lse, float* rowloss,
                               float* sa, float* sb, hipStream_t s);
// dZ chunk: rows [r0, r0+R) x vocab [c0, c0+Vc) of coef * (softmax - onehot), into
// staging [R, ldz] (dtype), zero past V.
hipError_t launch_ce_bwd_dz(int dtype, CeGemmShape t, const void* h, const void* W,
                            const int32_t* labels, const float* lse, const float* coef, int r0,
                            int R, int d, int c0, int Vc, int V, void* dz, int ldz, const int* gate,
                            hipStream_t s);
// Row scales of the label-referenced dH epilogue; all null for the plain dZ chunks.
struct CeRowScale {
  const float* sa = nullptr;
  const float* sb = nullptr;
  const int32_t* labels = nullptr;
};
// dH rows [r0, r0+R) (+)= staged chunk . W[c0 : c0+K]: f32 path reads W [V, d]; bf16 path reads
// WT [d, Vp]. first: no accumulator read; last: write grad (dtype) instead of acc (f32), with
// the row scales when rs.sa is set (bf16 only).
hipError_t launch_ce_bwd_dh(int dtype, CeGemmShape t, const void* dz, int ldz, const void* W,
                            const void* WT, int Vp, int r0, int R, int d, int c0, int K, int V,
                            float* acc, void* grad, bool first, bool last, const CeRowScale& rs,
                            const int* gate, hipStream_t s);

// ---- LoRA ------------------------------------------------------------------------------
constexpr int kLoraBatch = 16;

struct LoraJob {
  const void* x;
  const void* dy;
  const void* A;
  const void* B;
  float* dA;
  float* dB;
  int64_t ut_off;    // workspace byte offset of s*U^T  [rp, rows_pad] (dtype)
  int64_t dut_off;   // workspace byte offset of s*(dy B)^T [rp, rows_pad] (dtype)
  int64_t pa_off;    // workspace byte offset of dA partials [splits, rp, d_in] f32
  int64_t pb_off;    // workspace byte offset of dB partials [splits, rp, d_out] f32
  int32_t rows, rows_pad, d_in, d_out, rank, rp, splits;
  float scale;
  int32_t b1_begin;  // first pass-1 block (U and dU row tiles)
  int32_t b2_begin;  // first pass-2 block (dA / dB column blocks x splits)
  int32_t b3_begin;  // first reduce block
  int32_t pad;
};

struct LoraBatch {
  int32_t count;
  int32_t pad;
  LoraJob j[kLoraBatch];
};

constexpr int kLoraRowTile = 128;   // pass-1 rows per block
constexpr int kLoraColTile = 64;    // pass-2 output columns per block
constexpr int kLoraTStep = 32;      // pass-2 contraction step over rows

hipError_t launch_lora_pass1(int dtype, const LoraBatch& b, int blocks, uint8_t* ws, hipStream_t s);
hipError_t launch_lora_pass2(int dtype, const LoraBatch& b, int blocks, uint8_t* ws, hipStream_t s);
hipError_t launch_lora_reduce(const LoraBatch& b, int blocks, uint8_t* ws, hipStream_t s);

}  // namespace attt
