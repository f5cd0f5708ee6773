// Kernel argument blocks and launchers (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pd {

// Gathered KV rows of one decode shard whose cache-row codes fit the kernel's
// LDS table; the host raises the shard count until every shard fits.
constexpr int kDecodeTableRows = 2048;

// bf16 tile engine geometry: query rows per wave (32 or 64), waves per
// workgroup and the number of K/V tiles resident in LDS (the one being multiplied, the previous
// one, and the rest streaming in).  Build-time tunables.
#ifndef PD_BF16_ROWS_PER_WAVE
#define PD_BF16_ROWS_PER_WAVE 32
#endif
#ifndef PD_BF16_WAVES
#define PD_BF16_WAVES (PD_BF16_ROWS_PER_WAVE == 32 ? 8 : 4)
#endif
#ifndef PD_BF16_STAGES
#define PD_BF16_STAGES 4
#endif
constexpr int kBf16RowsPerWave = PD_BF16_ROWS_PER_WAVE;
constexpr int kBf16Waves = PD_BF16_WAVES;
constexpr int kBf16Rows = kBf16RowsPerWave * kBf16Waves;
static_assert(kBf16RowsPerWave == 32 || kBf16RowsPerWave == 64, "32 or 64 query rows per wave");
constexpr int kBf16Stages = PD_BF16_STAGES;
static_assert(kBf16Waves == 4 || kBf16Waves == 8, "4 or 8 waves per workgroup");
static_assert(kBf16Stages >= 3 && kBf16Stages <= 4, "3 or 4 stages");

// Stage (a).  Element pointers are bf16 bit patterns (uint16_t) or fp32.
struct PrefillArgs {
  const uint16_t *q_pre, *k_pre, *v_pre, *q_qm, *k_qm, *v_qm;
  uint16_t *o, *k_cache, *v_cache;
  float* part_i;   // [B][N][Hq][C]  per-head mass of content row j on the query columns
  float* lse_q;    // [B][N][Hq][Lq] log2-domain LSE of the query rows
  float* qm_mass;  // [B][N][Hq][Lq+Lm] mass of each q/m row on the C content columns, or nullptr
  float* km_part;  // bf16: [B][N][Hkv][n_qt*G][d] content-key sums of each cache-writing workgroup
  int B, N, C, Lq, Lm, Hq, Hkv, G, Sc;
  int n_qt, n_kvt, total;
  int qm_per_chunk;
  int out_f32;       // o is fp32 instead of the input element type
  float scale_log2;  // softmax scale * log2(e)
};

struct EscoreArgs {
  const uint16_t *q_qm, *k_cache;
  const float *part_i, *lse_q;
  float* part_io;    // bf16 path: per-head sums [B][N][Hq][C], updated in place (same buffer as part_i)
  float* tok_score;
  int B, N, C, Lq, Lm, Hq, Hkv, G, n_cb, total, qm_per_chunk;
  int q2c;           // 1: only the query rows' mass on the token (query-to-chunk score)
  float scale_log2;
};

// Stage (c).
struct DecodeArgs {
  const uint16_t *q_dec, *k_dec, *v_dec, *k_cache, *v_cache, *k_static, *v_static;
  const int32_t *chunk_idx, *tok_slot;
  void* o_dec;       // element type of the call
  float* lse_dec;    // natural-log LSE or nullptr (only when S == 1)
  float* o_part;     // [S][B][Hq][Ld][D] shard outputs (normalised), S > 1
  float* lse_part;   // [S][B][Hq][Ld] log2-domain shard LSE, S > 1
  int B, N, C, Hq, Hkv, G, Ld, Ls, K, Bt, n_static, S;
  int n_sel;         // prefix rows per (sequence, KV head): K*(1+Bt) gathered, or the compact count
  int compact;       // 1: prefix rows j < n_sel are rows of k_cache/v_cache laid out [B][Hkv][n_sel][D]
  int n_qt, total;
  int out_f32;       // o_dec is fp32 instead of the input element type
  float scale_log2;
};

hipError_t launch_prefill_bf16(const PrefillArgs& a, int head_dim, hipStream_t s);
hipError_t launch_escore_bf16(const EscoreArgs& a, int head_dim, hipStream_t s);
hipError_t launch_decode_bf16(const DecodeArgs& a, int head_dim, hipStream_t s);

hipError_t launch_prefill_f32(const PrefillArgs& a, int head_dim, hipStream_t s);
hipError_t launch_escore_f32(const EscoreArgs& a, int head_dim, hipStream_t s);
hipError_t launch_decode_f32(const DecodeArgs& a, int head_dim, hipStream_t s);

// Generic (both element types).
// Chunk cache copy (fp32 path; the bf16 prefill writes the cache itself).
hipError_t launch_cache_copy(const void* k_pre, const void* v_pre, void* k_cache, void* v_cache,
                             int B, int N, int C, int Hkv, int head_dim, int elem_bytes, hipStream_t s);
hipError_t launch_key_mean(const void* k_cache, float* key_mean, int B, int N, int C, int Hkv,
                           int head_dim, bool bf16, hipStream_t s);
hipError_t launch_merge(const float* o_part, const float* lse_part, void* o_dec, float* lse_dec,
                        int S, int B, int Hq, int Ld, int head_dim, bool bf16, hipStream_t s);

// Stage (b).
struct SelectArgs {
  const void* q_dec;
  const float* key_mean;
  const int32_t* tok_rank;
  float* partial;   // [B][N][Hq*NS] workspace: per (head, row split) chunk-score terms
  float* chunk_score;  // [B][N] or nullptr
  int32_t *chunk_idx, *tok_slot;
  int B, N, C, Hq, Hkv, G, Ld, D, K, Bt, NS;
  int q_rows, q_row0, q_bstride;   // rows averaged into the mean query: rows q_row0.. of q_bstride per sequence
  bool bf16;
  float scale;
};
hipError_t launch_score_select(const SelectArgs& a, hipStream_t s);
hipError_t launch_gather_selected(const void* k_cache, const void* v_cache, const int32_t* chunk_idx,
                                  const int32_t* tok_slot, void* k_sel, void* v_sel, int B, int N, int C, int Hkv,
                                  int K, int Bt, int row_bytes, hipStream_t s);
hipError_t launch_mfma_rate(int n_workgroups, int iters, float* sink, hipStream_t s);

// Full-mask cache construction: joint rows [kept rows ; query rows] per sequence.
struct JointArgs {
  const void *q_pre, *k_cache, *v_cache, *q_qm, *k_qm, *v_qm;
  const int32_t *chunk_idx, *tok_slot;
  void *q_joint, *k_joint, *v_joint;
  void *k_pref, *v_pref;   // optional [B][Hkv][Lj][d] copies of K, V (NULL: skipped)
  int B, N, C, Lq, Lm, Hq, Hkv, G, D, K, Bt, Lj, qm_per_chunk, elem_bytes;
  double rope_base;   // 0: no rotation
};
hipError_t launch_gather_joint(const JointArgs& a, hipStream_t s);
hipError_t launch_token_rank(const float* tok_score, int32_t* tok_rank, int B, int N, int C, hipStream_t s);
// e = sum over the H_q heads of the per-head sums (fixed order), then the ranks.
hipError_t launch_head_sum_rank(const float* per_head, float* tok_score, int32_t* tok_rank, int B, int N, int Hq,
                                int C, const float* km_part, float* key_mean, int Hkv, int D, int km_slots,
                                hipStream_t s);
hipError_t launch_chunk_score(const float* qm_mass, float* chunk_score, int B, int N, int Hq, int Lq, int Lm,
                              hipStream_t s);
hipError_t launch_select_ranked(const float* chunk_score, int lowest, const int32_t* tok_rank, int32_t* chunk_idx,
                                int32_t* tok_slot, int B, int N, int C, int K, int Bt, hipStream_t s);
int select_row_splits(int Ld);

}  // namespace pd
