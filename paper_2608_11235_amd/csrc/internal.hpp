// Host-side launch wrappers shared by the runtime (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cora {

// ---- weight init ------------------------------------------------------------------------
// Physical row of logical row r: 0 identity (+row_offset), 1 gate half and 2 up half of
// the 32-row interleaved gate/up matrix.
// 3: rows of q or k heads stored pair-interleaved within each head of hd rows (logical
// j < hd/2 at 2j, logical j + hd/2 at 2j + 1), after row_offset.
enum RowMap { ROW_IDENTITY = 0, ROW_GATE = 1, ROW_UP = 2, ROW_ROPE_PAIR = 3 };
hipError_t launch_init_bf16(uint16_t* dst, uint64_t seed, uint64_t tensor_id, int64_t rows,
                            int64_t cols, int64_t ld, int row_map, int64_t row_offset, double std_dev,
                            int head_dim, hipStream_t s, bool packed = false);
hipError_t launch_init_f32(float* dst, uint64_t seed, uint64_t tensor_id, int64_t n, double std_dev,
                           int pair_head_dim, hipStream_t s);
// physical position of logical index j inside a head of hd pair-interleaved rows
__host__ __device__ inline int rope_pair_pos(int j, int hd) { return j < hd / 2 ? 2 * j : 2 * (j - hd / 2) + 1; }
hipError_t launch_fill_f32(float* dst, float v, int64_t n, hipStream_t s);

// ---- elementwise ------------------------------------------------------------------------
hipError_t launch_embed(const int32_t* tokens, const uint16_t* E, float* h, int M, int d, int V,
                        hipStream_t s);
// out[j] = rmsnorm(h[src(j)]) with src(j) = j (mode 0), or for j = b * n_rows + r:
// b * L + row_begin + r (mode 1), b * L + lo_b + r with lo_b the active block start (mode 2).
struct RowSel {
  int mode, L, n_rows, row_begin, prompt_len, block_len, n_blocks;
  const int32_t* block_idx;
};
hipError_t launch_rmsnorm(const float* h, const float* w, uint16_t* out, int rows, int d,
                          float eps, RowSel sel, hipStream_t s);
// h[r, :] += part[0][r, :] + ... + part[splits-1][r, :] (partials [splits][rows][d], summed in
// split order), then, when out is not null, out[r, :] = bf16(rmsnorm(h[r, :]) * w).
// d % 4 == 0 and d <= RESIDUAL_NORM_MAX_D.
constexpr int RESIDUAL_NORM_MAX_D = 8192;
hipError_t launch_residual_norm(float* h, const float* part, int splits, int rows, int d,
                                const float* w, uint16_t* out, float eps, hipStream_t s);
hipError_t launch_state_init(const int32_t* prompt, int B, int P, int G, int mask_id,
                             int32_t* tokens, uint8_t* unresolved, int32_t* prev, int32_t* persist,
                             int32_t* block_idx, int32_t* step_idx, int32_t* passes, int n_blocks,
                             hipStream_t s);
// decode-state rows (device arrays of one state)
struct DecodeRows {
  int32_t* tokens; uint8_t* unresolved; int32_t* prev; int32_t* persist;
  int32_t* block_idx; int32_t* step_idx; int32_t* passes;
};
// dst row i <- src row map[i], i < n
hipError_t launch_gather_state(const DecodeRows& src, const DecodeRows& dst, const int32_t* map,
                               int n, int L, int n_blocks, hipStream_t s);
// out_tokens / out_passes row orig[i] <- tokens / passes row rows[i], i < n
hipError_t launch_scatter_rows(const int32_t* tokens, const int32_t* passes, const int32_t* rows,
                               const int32_t* orig, int n, int L, int n_blocks,
                               int32_t* out_tokens, int32_t* out_passes, hipStream_t s);

// ---- GEMM: C[M, N] = A[M, K] . W[N, K]^T, bf16 in, fp32 accumulate ---------------------
enum GemmEpi {
  EPI_BF16 = 0, EPI_ADD_F32 = 1, EPI_SWIGLU = 2, EPI_QKV_ROPE = 3, EPI_PART_F32 = 4, EPI_TOP1 = 5
};
// EPI_TOP1: no C; per row and wavefront column range, the (max, lowest arg max, sum of
// exp(l - max)) of the logits EPI_BF16 would write (bias none, then * scale, rounded to
// bf16), mask_id and columns past N left out, at part_*[row * n_parts + p] with
// p = column range index in vocab order (gemm_top1_parts ranges per row).
// EPI_PART_F32: split s of the K loop stores its fp32 partial product to
// ((float*)C)[s * M * ldc + row * ldc + col]; the partials are folded in by a later kernel
// (launch_residual_norm), so the GEMM itself takes no tickets.
// EPI_QKV_ROPE: columns [0, H*hd) are q heads, then Hkv*hd k heads, then Hkv*hd v heads;
// q and k weight rows are pair-interleaved per head (ROW_ROPE_PAIR).  Adds the bias,
// rotates q and k (rotate-half RoPE at position row % L), and writes q [B, H, Ls, hd],
// k [B, Hkv, Ls, hd] in the interleaved dim order and v transposed vt [B, Hkv, hd, Ls].
struct QkvOut {
  uint16_t *q, *k, *vt;
  const float *cos_t, *sin_t;  // [Ls, hd/2]
  int L, Ls, n_heads, n_kv_heads, head_dim;
};
struct GemmArgs {
  const uint16_t* A; int64_t lda;
  const uint16_t* W; int64_t ldw;
  int M, N, K;
  void* C; int64_t ldc;
  const float* bias;   // EPI_BF16: per-column bias (or null)
  float scale;         // EPI_BF16: multiplier after the bias
  int splits;          // set by launch_gemm from the plan
  QkvOut qkv;          // EPI_QKV_ROPE destinations
  bool w_packed;       // W in 64 x 64 blocks (N % 64 == 0, K % 64 == 0), see pack layout
  // EPI_TOP1 outputs
  float* part_m; float* part_s; int* part_arg;
  int n_parts, mask_id;
};
struct GemmPlan {
  int cfg, tiles, splits;
  size_t ws_floats;    // EPI_PART_F32 partial floats (splits * M * N) when splits > 1
};
// Whole-K plan for any epilogue; split plan (EPI_PART_F32 when splits > 1, else any
// epilogue) never needs more than gemm_ws_floats_bound(num_cus) partial floats.  With
// splits > 0 the split plan keeps that split count (it must divide K / 64 into runs of >= 8
// slices) and only picks the tile config; the split count alone decides the summation order
// of an output, the tile config does not.
GemmPlan gemm_plan(int M, int N, int K, int num_cus);
GemmPlan gemm_plan_split(int M, int N, int K, int num_cus, int splits = 0);
GemmPlan gemm_plan_cfg(int M, int N, int K, int cfg, int splits);
int gemm_num_cfgs();
inline size_t gemm_ws_floats_bound(int num_cus) { return (size_t)2 * num_cus * 256 * 256; }
// ev_start / ev_stop (optional): stamped with the kernel's start and end by the dispatch
hipError_t launch_gemm(int epi, const GemmArgs& a, const GemmPlan& p, hipStream_t s,
                       hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);
// EPI_TOP1 partials per row of a plan (column ranges of TN x 32 over the N tiles)
int gemm_top1_parts(const GemmPlan& p, int N);
// EPI_PART_F32 partials [splits][M][N] of the QKV projection -> the EPI_QKV_ROPE outputs.
hipError_t launch_qkv_finish(const float* part, int splits, int M, int N, const float* bias,
                             const QkvOut& o, hipStream_t s);

// ---- LM head for few rows (M <= 64) ------------------------------------------------------
struct LmHeadArgs {
  const uint16_t* A; int64_t lda;  // [M, K] normalised rows
  const uint16_t* Wp;              // vocab projection [N, K] in the packed layout
  int M, N, K;
  float scale;                     // logit scale, applied before the bf16 rounding
  uint16_t* logits; int64_t ldc;   // logits mode: [M, N] bf16
  // top-1 mode: per row, partial statistics of each 128-entry vocab range ([M][n_parts])
  float* part_m; float* part_s; int* part_arg;
  int n_parts;                     // set by launch_lm_head
  int mask_id;                     // left out of the top-1 statistics
};
constexpr int LM_HEAD_FUSED_MAX_ROWS = 64;
int lm_head_parts(int N);
// packed copy of the vocab projection (written once, read by launch_lm_head)
size_t lm_head_packed_elems(int N, int K);
hipError_t launch_pack_lm_head(const uint16_t* W, uint16_t* packed, int N, int K, hipStream_t s);
bool lm_head_supported(int M, int N, int K, int64_t lda);
hipError_t launch_lm_head(const LmHeadArgs& a, bool top1, hipStream_t s);
// rows are scored like launch_vocab_top1: row r of batch row b (n_rows per batch row) goes to
// top1/conf[b * out_ld + out_off + r]
hipError_t launch_top1_merge(const LmHeadArgs& a, int n_rows, int out_ld, int out_off,
                             int32_t* top1, float* conf, hipStream_t s);
// the same merge for M rows of n_parts partials each (EPI_TOP1 GEMM output)
hipError_t launch_top1_merge_parts(const float* pm, const float* ps, const int* pa, int n_parts,
                                   int M, int n_rows, int out_ld, int out_off, int32_t* top1,
                                   float* conf, hipStream_t s);

// ---- attention ---------------------------------------------------------------------------
// The key range is split into parts (merged in part order) by the grid of plan_B rows
// (plan_B >= B), so a row's output does not depend on how many rows share the launch.
hipError_t launch_attention(const uint16_t* q, const uint16_t* k, const uint16_t* vt,
                            uint16_t* out, int B, int L, int Ls, int H, int Hkv, int hd,
                            int plan_B, int num_cus, hipStream_t s);

// ---- vocab / gate -------------------------------------------------------------------------
// Logits rows r of batch row b (row-major [B, n_rows, V]) score canvas position
// row_begin + r (row_begin >= 0) or lo_b + r (row_begin < 0, lo_b = active block start).
// Their top-1 / confidence go to top1/conf[b * out_ld + out_off + r], so a region can be
// scored in chunks into one [B, out_ld] array.
struct VocabGateArgs {
  const uint16_t* logits; int n_rows; int row_begin; int V; int mask_id;
  int32_t* tokens; uint8_t* unresolved; int32_t* prev_top1; int32_t* persist;
  int32_t* block_idx; int32_t* step_idx; int32_t* top1; float* conf; uint8_t* decision;
  int32_t* done; int32_t* passes;
  int B, L, prompt_len, block_len, steps_per_block, n_blocks;
  int k_transfer;  // >= 0 fixed k, < 0: schedule
  float delta_p; int m_req; int gate_enabled;
  int persist_scope;  // 0 BLOCK, 1 GLOBAL (every scored unresolved position, no block reset)
  int out_ld, out_off;
  int eos_enabled, eos_id;  // EOS-aware controller
};
// top-1 and confidence of every logits row
hipError_t launch_vocab_top1(const VocabGateArgs& a, hipStream_t s);
// The same with each row's vocabulary split into `parts` consecutive ranges, one workgroup
// each, whose (max, sum, lowest arg max) partials go to pm / ps / pa [rows * parts] (caller
// memory, fully overwritten) and are folded in vocab order by k_top1_merge.  top1 agrees
// with launch_vocab_top1 bit for bit; conf differs only in the fp32 summation order.
struct VocabSplit {
  int parts, chunks;  // chunks: set by the launcher (16-byte chunks, or entries, per part)
  float* pm; float* ps; int* pa;
};
// parts for `rows` rows: ~4 workgroups per CU, each part >= 1024 chunks, rows * parts <=
// max_partials; 0 when even one part per row does not fit
int vocab_split_parts(int rows, int V, int num_cus, int64_t max_partials);
hipError_t launch_vocab_top1_split(const VocabGateArgs& a, const VocabSplit& sp, hipStream_t s);
// decision rules per batch row, reading the scores of rows [row_begin, row_begin + n_rows)
// (n_rows == out_ld) or of the active block (row_begin < 0)
hipError_t launch_gate_rules(const VocabGateArgs& a, hipStream_t s);

}  // namespace cora
