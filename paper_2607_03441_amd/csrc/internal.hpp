// Host-side interfaces between the C ABI layer (api.cpp) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace attt {

typedef uint16_t bf16_t;  // raw bfloat16 bits

// ---- kernel timing ---------------------------------------------------------------------
enum KernelId {
  K_NGRAM_COUNT = 0,
  K_NGRAM_WEIGHT,
  K_NGRAM_TABLE,
  K_CE_FWD,
  K_CE_LABEL,
  K_CE_ROW_REDUCE,
  K_CE_LOSS,
  K_CE_HEAD_T,
  K_CE_BWD_DZ,
  K_CE_BWD_DH,
  K_CE_GUARD,
  K_LORA_U,
  K_LORA_DADB,
  K_LORA_REDUCE,
  K_NGRAM_SET,
  K_NGRAM_SET_WEIGHT,
  K_LORA_SGD,
  K_CE_FUSED,
  K_REP_COUNT,
  K_REP_REDUCE,
  K_ATTN_FWD,
  K_ATTN_DKDV,
  K_ATTN_DQ,
  K_LORA_FWD,
  K_LORA_SWAP,
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
  int64_t part_global;         // index of this partition in the canon / list arrays
  int32_t hist_ngrams;         // history n-gram starts of the episode: max(0, H_e - n + 1)
  int32_t q0;                  // first query start of this partition, relative to the episode
  int32_t qn;                  // query starts in this partition, 1 .. kQMax
  int32_t slots;               // LDS table size, power of two >= 8 * qn (at most 32768)
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
  int64_t part_base;   // canon row of the episode's first partition
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

// The allocation-free n-gram entry point keeps its partial counts in a static device array of
// this many bytes (2048 rows of kQMax 16-bit counts); ngram_scratch gives its address on the
// current device.
constexpr size_t kNgramScratchBytes = (size_t)16 << 20;  // ATTT_NGRAM_NOALLOC_SCRATCH_BYTES
hipError_t ngram_scratch(void** ptr);

size_t ngram_count_lds(int slots, int n);
// canon [partitions][kQMax] u16: canonical query position of every query position;
// list [partitions][kQMax] (table slot or 0xFFFFFFFF for a repeat, entry) per query position
hipError_t launch_ngram_table(const NgramPartBatch& b, int max_slots, const int32_t* tokens, int n,
                              uint16_t* canon, uint2* list, hipStream_t s);
hipError_t launch_ngram_count(const NgramPartBatch& b, int total_blocks, int max_slots,
                              const int32_t* history, const int32_t* tokens, const uint2* list, int n,
                              uint16_t* partial, hipStream_t s);
hipError_t launch_ngram_weight(const NgramEpBatch& b, int total_blocks, int n, float w_min,
                               const uint16_t* partial, const uint16_t* canon, uint32_t* exposure,
                               float* weights, hipStream_t s);

// ---- update-text repetition (Eq. 6-7) ------------------------------------------------------
constexpr int kRepSlots = 16384;        // entries of each LDS word set of the count kernel
constexpr int kRepPartWords = 4096;     // words per hash partition the host plans for (load <= 1/4)
struct RepEp {
  int64_t text0;      // first text of the episode (index into the text offsets)
  int64_t wg_global;  // first count record of the episode ([pair][part] order, 4 ints each)
  int64_t pair_base;  // first pair of the episode in pair_counts
  int32_t ntexts;     // texts of the episode, >= 1; the last is the candidate
  int32_t parts;      // hash partitions per pair
  int32_t wg_begin;   // first count-kernel workgroup of the episode within the launch
  int32_t ep;         // episode index (outputs)
};
struct RepBatch {
  int32_t count;
  int32_t pad;
  RepEp e[kEpBatch];
};
hipError_t launch_rep_count(const RepBatch& b, int total_wgs, const int32_t* words, const int64_t* toff,
                            int32_t* counts, hipStream_t s);
hipError_t launch_rep_reduce(const RepBatch& b, const int32_t* counts, double tau, double* rho, double* nu,
                             int32_t* skip, int32_t* best, int32_t* pair_counts, hipStream_t s);

// ---- attention-block backward -----------------------------------------------------------------
struct AttnArgs {
  const bf16_t* q;     // [N][heads][128]
  const bf16_t* k;     // [N][kv_heads][128]
  const bf16_t* v;
  const bf16_t* dout;  // [N][heads][128]
  bf16_t* dq;
  bf16_t* dk;
  bf16_t* dv;
  float* lse;          // [heads][N]
  float* dsum;         // [heads][N]
  int32_t N, heads, kv_heads;
  float scale;
};
struct AttnEp {
  int64_t row0;     // first row of the episode
  int32_t L;        // rows
  int32_t blocks;   // 64-row blocks
  int32_t wg_begin; // first workgroup of the episode within the launch
  int32_t pad;
};
struct AttnBatch {
  int32_t count;
  int32_t pad;
  AttnEp e[kEpBatch];
};
// kernel 0: forward statistics, 1: dK and dV, 2: dQ
hipError_t launch_attn(int kernel, const AttnArgs& a, const AttnBatch& b, int wgs, hipStream_t s);

// ---- persistent n-gram set ---------------------------------------------------------------
struct NgramSetJob {
  void* set;         // the episode's set buffer
  int64_t tok_base;  // first token of the episode's x in `tokens`
  int32_t L;         // tokens of x
  int32_t block_begin;
};

struct NgramSetBatch {
  int32_t count;
  int32_t pad;
  NgramSetJob j[kEpBatch];
};

size_t ngram_set_bytes(int64_t slots, int n);
hipError_t launch_ngram_set_init(const NgramSetBatch& b, int64_t slots, int n, hipStream_t s);
hipError_t launch_ngram_set_append(const NgramSetBatch& b, int blocks, const int32_t* tokens, int64_t slots,
                                   int64_t capacity, int n, hipStream_t s);
hipError_t launch_ngram_set_weights(const NgramSetBatch& b, int blocks, const int32_t* tokens, int64_t slots,
                                    int n, float w_min, uint32_t* exposure, float* weights, hipStream_t s);

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
// Rows [r0, r0+R): sigma, lse, row loss and the dH row scales (sa, sb).
hipError_t launch_ce_row_final(int r0, int R, const float* sig_part, int n_vb, const float* label_logit,
                               const float* weights, const float* coef, float* lse, float* rowloss,
                               float* sa, float* sb, hipStream_t s);
// float32 backward: dZ chunk, rows [r0, r0+R) x vocab [c0, c0+Vc) of coef * (softmax - onehot)
// into staging [R, ldz], zero past V; then dH rows [r0, r0+R) (+)= dZ chunk . W[c0 : c0+K]
// (first: overwrite).
hipError_t launch_ce_bwd_dz(const float* h, const float* W, const int32_t* labels, const float* lse,
                            const float* coef, int r0, int R, int d, int c0, int Vc, int V, float* dz, int ldz,
                            hipStream_t s);
hipError_t launch_ce_bwd_dh(const float* dz, int ldz, const float* W, int r0, int R, int d, int c0, int K, int V,
                            float* grad, bool first, hipStream_t s);

// Fused bf16 backward (ce_fused.hip): one persistent cooperative grid of 8 x kCeTeam workgroups,
// one per CU, in XCD teams of kCeTeam producers and consumers sharing a ring of bf16 tiles.
constexpr int kCeTeam = 32;
struct CeFusedArgs {
  const bf16_t* h;            // [N, d]
  const bf16_t* W;            // [V, d]
  const bf16_t* WT;           // [d, Vp], columns V .. Vp-1 zero
  const int32_t* labels;      // [N]
  const float* label_logit;   // [N]  label mode
  const float* lse;           // [N]  exact mode
  const float* coef;          // [N]  w / L_e
  float* sig_part;            // [N, nv] per-(row, vocab tile) sums of e, label mode
  bf16_t* grad;               // [N, d]
  uint8_t* ring;              // 8 x slots tiles of 256 x 256 bf16
  int* sync;                  // zeroed sync area of ce_fused_sync_ints(slots) ints
  int* gate;                  // guard flag: set on overflow (label mode); exact mode runs only if set
  uint64_t limit;             // bound of every wait, ticks of the 100 MHz wall clock
  int N, d, V, Vp;
  int nv;                     // vocabulary tiles of 256
  int row_tiles;              // row tiles of 256
  int slices;                 // d-slices of 256
  int consumers;              // consumers per team; producers = kCeTeam - consumers
  int passes;                 // ceil(slices / consumers): the row tile's tiles are made once per pass
  int ksplit;                 // consumers per d-slice (F): part f takes vocabulary tiles f, f + F, ...
                              // (F > 1 only with one pass and consumers = slices x F)
  float* partial;             // F > 1: [8 teams][slices][F - 1][256 x 256] float32 partial sums
  int slots;                  // ring slots per XCD
  int items_max;              // items of the busiest team, rounded up to a multiple of 4
};
size_t ce_fused_ring_bytes(int slots);
int ce_fused_sync_ints(int slots, int items_max);
hipError_t launch_ce_sync_clear(int* sync, int n, hipStream_t s);
hipError_t launch_ce_fused(bool label, const CeFusedArgs& a, hipStream_t s);
hipError_t launch_ce_fused_status(const int* sync, int* gate, hipStream_t s);
hipError_t launch_ce_fused_nan(const int* sync, float* loss, int E, float* lse, int N, void* grad, int64_t nd,
                               hipStream_t s);

// ---- LoRA ------------------------------------------------------------------------------
constexpr int kLoraRowTile = 128;  // row padding of the transposed pass-1 results
constexpr int kLoraP1Rows = 64;    // pass-1 rows per workgroup (16 per wave)
constexpr int kLoraKBlock = 128;   // pass-1 contraction step
constexpr int kLoraColTile = 64;   // pass-2 output columns per workgroup
constexpr int kLoraTStep = 64;     // pass-2 rows per step
constexpr int kLoraMaxTiles = 4;   // rank tiles of 16 per job (64 ranks)
constexpr int kLoraJobBatch = 16;  // jobs per launch (kernel-argument descriptors)

// Pass 1: rows of `src` [rows, kdim] times up to four rank tiles of row-major adapter
// operands [rank, kdim] (A, or B^T in the workspace); tile t writes scale * (src op^T)^T at
// workspace offset out_off: float32 [16, rows_pad], or bf16 planes hi, lo [2][16, rows_pad].
struct LoraP1Tile {
  const void* op;   // first row of the tile in its operand
  int64_t out_off;
  float scale;
  int32_t valid;    // operand rows in the tile (rank - 16 t, at most 16); the rest read as zero
};
struct LoraP1Job {
  const void* src;
  int32_t rows, rows_pad, kdim, nt;
  int32_t b_begin, pad;
  LoraP1Tile t[kLoraMaxTiles];
};

// Pass 2: out[c, k] = sum_t L[c, t] src[t, k] per rank tile; L is a pass-1 result at lt_off
// (bf16: planes hi and lo, [2][16, rows_pad]; float32: [16, rows_pad]); float32 partials
// [splits, 16, cols] at part_off.
struct LoraP2Tile {
  int64_t lt_off;
  int64_t part_off;
};
struct LoraP2Job {
  const void* src;
  int32_t rows, rows_pad, cols, splits, nt;
  int32_t b_begin;
  LoraP2Tile t[kLoraMaxTiles];
};

// Reduce: dA [rank, d_in] += sum of the dA partials ([tiles, sa, 16, d_in] at pa_off), and
// dB [d_out, rank] += the transposed sum of the dB partials ([tiles, sb, 16, d_out] at pb_off).
struct LoraRedJob {
  float* dA;
  float* dB;
  int64_t pa_off, pb_off;
  int32_t rank, d_in, d_out, sa, sb;
  int32_t b_begin;
};

// B [d_out, rank] -> B^T [rp, d_out] at bt_off.
struct LoraBTJob {
  const void* B;
  int64_t bt_off;
  int32_t rank, rp, d_out;
  int32_t b_begin;
};

template <class J, int Cap = kLoraJobBatch>
struct LoraBatchOf {
  static constexpr int kCap = Cap;
  int32_t count;
  int32_t pad;
  J j[Cap];
};
using LoraP1Batch = LoraBatchOf<LoraP1Job>;
using LoraP2Batch = LoraBatchOf<LoraP2Job>;
using LoraRedBatch = LoraBatchOf<LoraRedJob>;
using LoraBTBatch = LoraBatchOf<LoraBTJob>;

// Adapter step: param [n] -= lr * grad [n] (float32), optional bf16 copy, optional grad reset.
struct LoraSgdJob {
  float* param;
  float* grad;
  uint16_t* param_bf16;  // nullable
  int64_t n;
  int32_t b_begin;
  int32_t pad;
};
using LoraSgdBatch = LoraBatchOf<LoraSgdJob>;
constexpr int kLoraSgdPerBlock = 1024;  // elements per workgroup (256 threads x 4)
hipError_t launch_lora_sgd(const LoraSgdBatch& b, int blocks, float lr, int zero_grad, hipStream_t s);

hipError_t launch_lora_bt(int dtype, const LoraBTBatch& b, int blocks, uint8_t* ws, hipStream_t s);
// nt: the largest rank-tile count of the batch's jobs (bf16 kernels are specialised on it)
hipError_t launch_lora_pass1(int dtype, int nt, const LoraP1Batch& b, int blocks, uint8_t* ws,
                             hipStream_t s);
hipError_t launch_lora_pass2(int dtype, const LoraP2Batch& b, int blocks, uint8_t* ws, hipStream_t s);
hipError_t launch_lora_reduce(const LoraRedBatch& b, int blocks, uint8_t* ws, hipStream_t s);

// ---- serving: grouped multi-adapter forward, adapter swap --------------------------------
// A job is a group of adapted projections reading one input x [rows, d_in] (one episode's
// rows; q, k and v of a layer together). Phase 1 computes U = x A^T for up to four units of
// 16 ranks; phase 2 adds scale-weighted U B^T into each projection's y [rows, d_out].
struct LoraFwdUnit {
  const void* A;    // first row of the unit in its problem's A [rank, d_in]
  float scale;
  int32_t valid;    // ranks in the unit (<= 16); the rest read as zero
};
struct LoraFwdOut {
  const void* B;    // [d_out, rank]
  void* y;          // [rows, d_out], updated in place
  int32_t d_out, rank;
  int32_t u0;       // first column of U that belongs to this projection
  int32_t pad;
};
struct LoraFwdJob {
  const void* x;
  int32_t rows, d_in;
  int32_t nu, no;   // units, projections
  int32_t rb;       // rows per workgroup: 64 (one wave per 16 rows) or 16 (the waves split d_in)
  int32_t kw;       // waves splitting d_in: 1, 4, or 8 (8-wave workgroups)
  int32_t ncs;      // column splits of the outputs (workgroups per row block)
  int32_t b_begin;  // first logical workgroup
  LoraFwdUnit u[kLoraMaxTiles];
  LoraFwdOut o[kLoraMaxTiles];
};
constexpr int kLoraFwdBatch = 16;
struct LoraFwdBatch {
  int32_t count;
  int32_t total;    // logical workgroups
  LoraFwdJob j[kLoraFwdBatch];
};
static_assert(sizeof(LoraFwdBatch) <= 3840, "kernel arguments");
// nu: the largest unit count of the batch's jobs; waves: 4, or 8 for jobs of at most 16 rows
// (kw = 8)
hipError_t launch_lora_fwd(int nu, int waves, const LoraFwdBatch& b, hipStream_t s);

// Swap: dst (bf16) = RN(src (float32)) for every tensor of the batch.
struct LoraSwapJob {
  const float* src;
  uint16_t* dst;
  int64_t n;
  int32_t b_begin;
  int32_t vec;      // src and dst 16-byte aligned
};
using LoraSwapBatch = LoraBatchOf<LoraSwapJob, 96>;  // 3 KiB of kernel arguments
static_assert(sizeof(LoraSwapBatch) <= 3840, "kernel arguments");
constexpr int kLoraSwapPerBlock = 2048;  // elements per workgroup (256 threads x 8)
hipError_t launch_lora_swap(const LoraSwapBatch& b, int blocks, hipStream_t s);

}  // namespace attt
