// C-ABI entry points: argument validation, workspace layout, launches.
// Everything here runs on the host; kernels are enqueued on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "pd.h"
#include "pd_kernels.h"

namespace {

thread_local std::string g_last_error;

pd_status fail(pd_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

pd_status ok() {
  g_last_error.clear();
  return PD_OK;
}

constexpr int kMaxChunks = 1024;
constexpr int kMaxChunkLen = 4096;
constexpr int kMaxSplits = 64;
constexpr int kMaxCompactRows = 1 << 20;   // prefix rows of a compact decode call
constexpr int kTargetWorkgroups = 256 * 8 / pd::kBf16Waves;  // two resident waves per SIMD on 256 CUs
constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

pd_status check_dims(const pd_dims* d) {
  if (!d) return fail(PD_ERR_NULL_PTR, "dims is NULL");
  if (d->batch < 1) return fail(PD_ERR_BAD_DIMS, "batch=%d must be >= 1", d->batch);
  if (d->n_chunks < 1 || d->n_chunks > kMaxChunks)
    return fail(PD_ERR_BAD_DIMS, "n_chunks=%d must be in 1..%d", d->n_chunks, kMaxChunks);
  if (d->chunk_len < 1 || d->chunk_len > kMaxChunkLen)
    return fail(PD_ERR_BAD_DIMS, "chunk_len=%d must be in 1..%d", d->chunk_len, kMaxChunkLen);
  if (d->q_len < 1) return fail(PD_ERR_BAD_DIMS, "q_len=%d must be >= 1", d->q_len);
  if (d->m_len < 0) return fail(PD_ERR_BAD_DIMS, "m_len=%d must be >= 0", d->m_len);
  if (d->dec_len < 1) return fail(PD_ERR_BAD_DIMS, "dec_len=%d must be >= 1", d->dec_len);
  if (d->n_heads_q < 1 || d->n_heads_kv < 1)
    return fail(PD_ERR_BAD_DIMS, "head counts %d/%d must be >= 1", d->n_heads_q, d->n_heads_kv);
  if (d->qm_per_chunk != 0 && d->qm_per_chunk != 1)
    return fail(PD_ERR_BAD_DIMS, "qm_per_chunk=%d must be 0 or 1", d->qm_per_chunk);
  if (d->out_fp32 != 0 && d->out_fp32 != 1)
    return fail(PD_ERR_BAD_DIMS, "out_fp32=%d must be 0 or 1", d->out_fp32);
  if (d->tok_score_dir != 0 && d->tok_score_dir != 1)
    return fail(PD_ERR_BAD_DIMS, "tok_score_dir=%d must be 0 or 1", d->tok_score_dir);
  if (d->n_heads_q % d->n_heads_kv != 0)
    return fail(PD_ERR_UNSUPPORTED, "n_heads_q=%d is not a multiple of n_heads_kv=%d", d->n_heads_q, d->n_heads_kv);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(PD_ERR_UNSUPPORTED, "head_dim=%d must be 64 or 128", d->head_dim);
  if (d->dtype != PD_BF16 && d->dtype != PD_FP32)
    return fail(PD_ERR_UNSUPPORTED, "dtype=%d is neither PD_BF16 nor PD_FP32", d->dtype);
  if (!(std::isfinite(d->sm_scale))) return fail(PD_ERR_BAD_DIMS, "sm_scale is not finite");
  // Grid sizes must fit one launch dimension.
  const long long sc = 1LL + d->chunk_len + d->q_len + d->m_len;
  if (sc > (1LL << 24) || d->dec_len > (1 << 24))
    return fail(PD_ERR_BAD_DIMS, "sequence length too large");
  // Kernels address rows inside one sequence's cache, chunk sequence or decode
  // block with 32-bit element offsets.
  if ((long long)d->n_chunks * d->n_heads_kv * (d->chunk_len + 1) * d->head_dim >= (1LL << 31))
    return fail(PD_ERR_BAD_DIMS, "one sequence's cache (n_chunks*n_heads_kv*(chunk_len+1)*head_dim) must stay below 2^31 elements");
  if (sc * std::max(d->n_heads_q, d->n_heads_kv) * d->head_dim >= (1LL << 31) ||
      (long long)d->dec_len * d->n_heads_q * d->head_dim >= (1LL << 31))
    return fail(PD_ERR_BAD_DIMS, "rows of one sequence exceed 2^31 elements");
  const long long grid = (long long)d->batch * d->n_chunks * d->n_heads_q * cdiv(sc, 64);
  if (grid >= (1LL << 31)) return fail(PD_ERR_BAD_DIMS, "problem too large for one launch");
  return PD_OK;
}

int elem_bytes(const pd_dims* d) { return d->dtype == PD_BF16 ? 2 : 4; }
float scale_of(const pd_dims* d) { return d->sm_scale > 0.f ? d->sm_scale : 1.0f / std::sqrt((float)d->head_dim); }

// --- workspace layouts -------------------------------------------------------
struct PrefillWs {
  size_t part_i, lse_q, qm_mass, km_part, total;
};
// Writer slots of the key-mean partial sums: one per (query tile, head of the
// KV group) of the bf16 prefill.
int km_slots(const pd_dims* d) {
  const long long sc = 1LL + d->chunk_len + d->q_len + d->m_len;
  return cdiv(sc, pd::kBf16Rows) * (d->n_heads_q / d->n_heads_kv);
}
PrefillWs prefill_ws(const pd_dims* d) {
  PrefillWs w;
  const size_t bnh = (size_t)d->batch * d->n_chunks * d->n_heads_q;
  const size_t bng = (size_t)d->batch * d->n_chunks * d->n_heads_kv;
  w.part_i = 0;
  w.lse_q = round_up(bnh * d->chunk_len * sizeof(float));
  w.qm_mass = w.lse_q + round_up(bnh * d->q_len * sizeof(float));
  w.km_part = w.qm_mass + round_up(bnh * (d->q_len + d->m_len) * sizeof(float));
  w.total = w.km_part + (d->dtype == PD_BF16 ? round_up(bng * km_slots(d) * d->head_dim * sizeof(float)) : 0);
  return w;
}

// Chunk-score terms [B][N][H_q * row splits]; sized for the larger of the two
// row sets a selection averages (L_d decode rows, or L_m pseudo-label rows).
size_t select_ws(const pd_dims* d) {
  const int rows = std::max(d->dec_len, std::max(d->m_len, 1));
  return round_up((size_t)d->batch * d->n_chunks * d->n_heads_q * pd::select_row_splits(rows) * sizeof(float));
}

int decode_qtiles(const pd_dims* d) {
  const int G = d->n_heads_q / d->n_heads_kv;
  return d->dtype == PD_BF16 ? cdiv((long long)G * d->dec_len, pd::kBf16Rows) : cdiv(d->dec_len, 64);
}
long long decode_units(const pd_dims* d) {
  return (long long)d->batch * (d->dtype == PD_BF16 ? d->n_heads_kv : d->n_heads_q) * decode_qtiles(d);
}

// Launch sizes that must fit one grid dimension: the decode (work items x
// shards), its Split-S merge (one thread per 4 output elements), and the
// chunk-score pass over `rows` query rows (sequence x head x 128-row split).
pd_status check_decode_grid(const pd_dims* d, int S) {
  const long long total = decode_units(d) * S;
  const long long merge = ((long long)d->batch * d->n_heads_q * d->dec_len * (d->head_dim / 4) + 255) / 256;
  if (total >= (1LL << 31) || (S > 1 && merge >= (1LL << 31)))
    return fail(PD_ERR_BAD_DIMS, "decode of batch=%d, dec_len=%d with %d shards is too large for one launch",
                d->batch, d->dec_len, S);
  return PD_OK;
}
pd_status check_select_grid(const pd_dims* d, int rows) {
  if ((long long)d->batch * d->n_heads_q * pd::select_row_splits(rows) >= (1LL << 31))
    return fail(PD_ERR_BAD_DIMS, "chunk scoring of batch=%d over %d query rows is too large for one launch",
                d->batch, rows);
  return PD_OK;
}

// Shard counts for a decode call whose KV has n_sel prefix rows per (sequence,
// KV head) ahead of the static and own rows.  Requested count: explicit, or
// chosen so that the decode grid fills the CUs while every shard keeps >= 4 KV
// tiles of 64 rows.  The bf16 kernel also needs every shard to fit its LDS row
// table (at most kDecodeTableRows rows, i.e. kDecodeTableRows/64 tiles),
// whatever n_static is.
int min_splits(const pd_dims* d, long long n_sel) {
  if (d->dtype != PD_BF16 || n_sel <= pd::kDecodeTableRows) return 1;
  const long long lkv_max = n_sel + d->q_len + d->m_len + d->dec_len;
  return cdiv(cdiv(lkv_max, 64), pd::kDecodeTableRows / 64);
}

int requested_splits(const pd_dims* d, long long n_sel, int num_splits) {
  int s = num_splits;
  if (s <= 0) {
    const long long lkv0 = n_sel + d->dec_len;
    const int max_by_len = std::max(1, cdiv(lkv0, 64) / 4);
    const int want = cdiv(kTargetWorkgroups, std::max(1LL, decode_units(d)));
    s = std::max(1, std::min(std::min(want, max_by_len), kMaxSplits));
  }
  return std::max(s, min_splits(d, n_sel));
}

int effective_splits(const pd_dims* d, long long n_sel, int n_static, int num_splits) {
  const long long lkv = n_sel + n_static + d->dec_len;
  const int tile = d->dtype == PD_BF16 ? 64 : 32;
  return std::max(1, std::min(requested_splits(d, n_sel, num_splits), cdiv(lkv, tile)));
}

long long n_sel_of(int top_k, int tok_budget) { return (long long)top_k * (1 + tok_budget); }

// The decode kernels address the static and own rows of a (sequence, KV head)
// as row * H_kv * d from a base shifted back by the prefix rows, in 32-bit
// element offsets: every KV row index of one call, times H_kv * d, must stay
// below 2^31.
pd_status check_decode_rows(const pd_dims* d, long long n_sel, long long n_static) {
  const long long rows = n_sel + n_static + d->dec_len;
  if (rows * d->n_heads_kv * d->head_dim >= (1LL << 31))
    return fail(PD_ERR_BAD_DIMS,
                "decode KV rows (n_sel=%lld + n_static=%lld + dec_len=%d) * n_heads_kv * head_dim must stay below 2^31",
                n_sel, n_static, d->dec_len);
  return PD_OK;
}

size_t decode_ws_bytes(const pd_dims* d, int S) {
  if (S <= 1) return 0;
  const size_t rows = (size_t)S * d->batch * d->n_heads_q * d->dec_len;
  return round_up(rows * d->head_dim * sizeof(float)) + round_up(rows * sizeof(float));
}

pd_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return PD_OK;
  if (!ws) return fail(PD_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if (!aligned16(ws)) return fail(PD_ERR_MISALIGNED, "workspace is not 16-byte aligned");
  if (have < need) return fail(PD_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return PD_OK;
}

#define PD_REQUIRE_PTR(p)                                               \
  do {                                                                  \
    if (!(p)) return fail(PD_ERR_NULL_PTR, "pointer '%s' is NULL", #p); \
    if (!aligned16(p)) return fail(PD_ERR_MISALIGNED, "pointer '%s' is not 16-byte aligned", #p); \
  } while (0)

#define PD_RETURN_IF(st)          \
  do {                            \
    pd_status _s = (st);          \
    if (_s != PD_OK) return _s;   \
  } while (0)

pd_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(PD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

const char* pd_version(void) { return "pd-mi355x 0.1 (gfx950)"; }

pd_status pd_mfma_rate_probe(int32_t n_workgroups, int32_t iters, float* sink, void* stream) {
  if (!sink) return fail(PD_ERR_NULL_PTR, "sink is NULL");
  if (n_workgroups < 1 || iters < 1 || n_workgroups > (1 << 20))
    return fail(PD_ERR_BAD_DIMS, "n_workgroups=%d must be in 1..2^20 and iters=%d >= 1", n_workgroups, iters);
  if (!aligned16(sink)) return fail(PD_ERR_MISALIGNED, "sink is not 16-byte aligned");
  return hip_status(pd::launch_mfma_rate(n_workgroups, iters, sink, (hipStream_t)stream), "mfma rate probe");
}

const char* pd_status_string(pd_status s) {
  switch (s) {
    case PD_OK: return "PD_OK";
    case PD_ERR_NULL_PTR: return "PD_ERR_NULL_PTR";
    case PD_ERR_BAD_DIMS: return "PD_ERR_BAD_DIMS";
    case PD_ERR_UNSUPPORTED: return "PD_ERR_UNSUPPORTED";
    case PD_ERR_MISALIGNED: return "PD_ERR_MISALIGNED";
    case PD_ERR_WORKSPACE: return "PD_ERR_WORKSPACE";
    case PD_ERR_HIP: return "PD_ERR_HIP";
  }
  return "PD_ERR_UNKNOWN";
}

const char* pd_last_error_message(void) { return g_last_error.c_str(); }

size_t pd_cache_bytes(const pd_dims* d) {
  if (check_dims(d) != PD_OK) return 0;
  return (size_t)d->batch * d->n_chunks * d->n_heads_kv * (d->chunk_len + 1) * d->head_dim * elem_bytes(d);
}

size_t pd_workspace_bytes(const pd_dims* d, int32_t top_k, int32_t tok_budget, int32_t num_splits, int32_t which) {
  if (check_dims(d) != PD_OK) return 0;
  switch (which) {
    case 0: return prefill_ws(d).total;
    case 1:
      if (check_select_grid(d, std::max(d->dec_len, std::max(d->m_len, 1))) != PD_OK) return 0;
      return select_ws(d);
    case 2: {
      if (top_k < 1 || tok_budget < 1 || num_splits < 0 || num_splits > kMaxSplits) return 0;
      if (check_decode_rows(d, n_sel_of(top_k, tok_budget), 0) != PD_OK) return 0;
      const int S = requested_splits(d, n_sel_of(top_k, tok_budget), num_splits);
      if (check_decode_grid(d, S) != PD_OK) return 0;
      return decode_ws_bytes(d, S);
    }
    default: return 0;
  }
}

int32_t pd_decode_splits(const pd_dims* d, int32_t top_k, int32_t tok_budget, int32_t n_static, int32_t num_splits) {
  if (check_dims(d) != PD_OK || top_k < 1 || tok_budget < 1 || num_splits < 0 || num_splits > kMaxSplits) return 0;
  return effective_splits(d, n_sel_of(top_k, tok_budget), n_static, num_splits);
}

pd_status pd_prefill_chunks(const pd_dims* d, const void* q_pre, const void* k_pre, const void* v_pre,
                            const void* q_qm, const void* k_qm, const void* v_qm, void* o, void* k_cache,
                            void* v_cache, float* tok_score, int32_t* tok_rank, float* key_mean, float* chunk_score,
                            void* workspace, size_t ws_bytes, void* stream) {
  PD_RETURN_IF(check_dims(d));
  PD_REQUIRE_PTR(q_pre);
  PD_REQUIRE_PTR(k_pre);
  PD_REQUIRE_PTR(v_pre);
  PD_REQUIRE_PTR(q_qm);
  PD_REQUIRE_PTR(k_qm);
  PD_REQUIRE_PTR(v_qm);
  PD_REQUIRE_PTR(o);
  PD_REQUIRE_PTR(k_cache);
  PD_REQUIRE_PTR(v_cache);
  PD_REQUIRE_PTR(tok_score);
  PD_REQUIRE_PTR(tok_rank);
  PD_REQUIRE_PTR(key_mean);
  if (chunk_score && !aligned16(chunk_score))
    return fail(PD_ERR_MISALIGNED, "pointer 'chunk_score' is not 16-byte aligned");
  const PrefillWs w = prefill_ws(d);
  PD_RETURN_IF(check_ws(workspace, ws_bytes, w.total));

  hipStream_t s = (hipStream_t)stream;
  const bool bf16 = d->dtype == PD_BF16;
  char* ws = (char*)workspace;
  pd::PrefillArgs a{};
  a.q_pre = (const uint16_t*)q_pre;
  a.k_pre = (const uint16_t*)k_pre;
  a.v_pre = (const uint16_t*)v_pre;
  a.q_qm = (const uint16_t*)q_qm;
  a.k_qm = (const uint16_t*)k_qm;
  a.v_qm = (const uint16_t*)v_qm;
  a.o = (uint16_t*)o;
  a.k_cache = (uint16_t*)k_cache;
  a.v_cache = (uint16_t*)v_cache;
  a.part_i = (float*)(ws + w.part_i);
  a.lse_q = (float*)(ws + w.lse_q);
  a.qm_mass = chunk_score ? (float*)(ws + w.qm_mass) : nullptr;
  a.km_part = (float*)(ws + w.km_part);
  a.B = d->batch;
  a.N = d->n_chunks;
  a.C = d->chunk_len;
  a.Lq = d->q_len;
  a.Lm = d->m_len;
  a.Hq = d->n_heads_q;
  a.Hkv = d->n_heads_kv;
  a.G = a.Hq / a.Hkv;
  a.Sc = 1 + a.C + a.Lq + a.Lm;
  a.qm_per_chunk = d->qm_per_chunk;
  a.out_f32 = d->out_fp32;
  a.scale_log2 = scale_of(d) * 1.4426950408889634f;
  a.n_qt = cdiv(a.Sc, bf16 ? pd::kBf16Rows : 64);
  a.n_kvt = cdiv(a.Sc, 64);
  a.total = a.B * a.N * a.Hq * a.n_qt;

  pd::EscoreArgs e{};
  e.q_qm = a.q_qm;
  e.k_cache = a.k_cache;
  e.part_i = a.part_i;
  e.part_io = a.part_i;
  e.lse_q = a.lse_q;
  e.tok_score = tok_score;
  e.B = a.B;
  e.N = a.N;
  e.C = a.C;
  e.Lq = a.Lq;
  e.Lm = a.Lm;
  e.Hq = a.Hq;
  e.Hkv = a.Hkv;
  e.G = a.G;
  e.n_cb = cdiv(a.C, 64);
  e.total = a.B * a.N * e.n_cb;
  e.qm_per_chunk = a.qm_per_chunk;
  e.q2c = d->tok_score_dir;
  e.scale_log2 = a.scale_log2;

  hipError_t err;
  if (bf16) {
    err = pd::launch_prefill_bf16(a, d->head_dim, s);
    if (err != hipSuccess) return hip_status(err, "prefill kernel");
    err = pd::launch_escore_bf16(e, d->head_dim, s);
    if (err != hipSuccess) return hip_status(err, "token-score kernel");
    err = pd::launch_head_sum_rank(a.part_i, tok_score, tok_rank, a.B, a.N, a.Hq, a.C, a.km_part, key_mean, a.Hkv,
                                   d->head_dim, km_slots(d), s);
    if (err != hipSuccess) return hip_status(err, "token-rank kernel");
  } else {
    err = pd::launch_prefill_f32(a, d->head_dim, s);
    if (err != hipSuccess) return hip_status(err, "prefill kernel");
    err = pd::launch_cache_copy(k_pre, v_pre, k_cache, v_cache, a.B, a.N, a.C, a.Hkv, d->head_dim, 4, s);
    if (err != hipSuccess) return hip_status(err, "cache copy kernel");
    err = pd::launch_escore_f32(e, d->head_dim, s);
    if (err != hipSuccess) return hip_status(err, "token-score kernel");
    err = pd::launch_token_rank(tok_score, tok_rank, a.B, a.N, a.C, s);
    if (err != hipSuccess) return hip_status(err, "token-rank kernel");
    err = pd::launch_key_mean(k_cache, key_mean, a.B, a.N, a.C, a.Hkv, d->head_dim, false, s);
    if (err != hipSuccess) return hip_status(err, "key-mean kernel");
  }
  if (chunk_score) {
    err = pd::launch_chunk_score(a.qm_mass, chunk_score, a.B, a.N, a.Hq, a.Lq, a.Lm, s);
    if (err != hipSuccess) return hip_status(err, "chunk-score kernel");
  }
  return ok();
}

pd_status pd_select_ranked(const pd_dims* d, int32_t top_k, int32_t tok_budget, const float* chunk_score,
                           int32_t lowest, const int32_t* tok_rank, int32_t* chunk_idx, int32_t* tok_slot,
                           void* stream) {
  PD_RETURN_IF(check_dims(d));
  if (top_k < 1 || top_k > d->n_chunks)
    return fail(PD_ERR_BAD_DIMS, "top_k=%d must be in 1..n_chunks=%d", top_k, d->n_chunks);
  if (tok_budget < 1 || tok_budget > d->chunk_len)
    return fail(PD_ERR_BAD_DIMS, "tok_budget=%d must be in 1..chunk_len=%d", tok_budget, d->chunk_len);
  if (lowest != 0 && lowest != 1) return fail(PD_ERR_BAD_DIMS, "lowest=%d must be 0 or 1", lowest);
  PD_REQUIRE_PTR(chunk_score);
  PD_REQUIRE_PTR(tok_rank);
  PD_REQUIRE_PTR(chunk_idx);
  PD_REQUIRE_PTR(tok_slot);
  return hip_status(pd::launch_select_ranked(chunk_score, lowest, tok_rank, chunk_idx, tok_slot, d->batch,
                                             d->n_chunks, d->chunk_len, top_k, tok_budget, (hipStream_t)stream),
                    "select kernel");
}

}  // extern "C"

// Scratch of pd_score_select_noalloc: one array per GPU holding the selection
// workspace (the chunk-score terms, fully rewritten by every call before the
// selection kernel reads them, so nothing needs clearing).  Host code never passes the array's name to a kernel:
// the address of each device's copy comes from hipGetSymbolAddress.
constexpr size_t kNoallocScratchBytes = 4u << 20;
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch[kMaxDevices];

// Device address of the current device's scratch, looked up once per device.
pd_status scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(PD_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(PD_ERR_UNSUPPORTED, "device %d is beyond the %d devices of the scratch table", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(PD_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return PD_OK;
}

// Shared by the selection entry points: sizes and pointers checked here, the
// mean query over `rows` rows starting at row0 of every bstride rows of q.
pd_status select_args(const pd_dims* d, int32_t top_k, int32_t tok_budget, const void* q, const float* key_mean,
                      const int32_t* tok_rank, int32_t* chunk_idx, int32_t* tok_slot, float* chunk_score,
                      pd::SelectArgs* a) {
  if (top_k < 1 || top_k > d->n_chunks)
    return fail(PD_ERR_BAD_DIMS, "top_k=%d must be in 1..n_chunks=%d", top_k, d->n_chunks);
  if (tok_budget < 1 || tok_budget > d->chunk_len)
    return fail(PD_ERR_BAD_DIMS, "tok_budget=%d must be in 1..chunk_len=%d", tok_budget, d->chunk_len);
  PD_REQUIRE_PTR(q);
  PD_REQUIRE_PTR(key_mean);
  PD_REQUIRE_PTR(tok_rank);
  PD_REQUIRE_PTR(chunk_idx);
  PD_REQUIRE_PTR(tok_slot);
  if (chunk_score && !aligned16(chunk_score))
    return fail(PD_ERR_MISALIGNED, "pointer 'chunk_score' is not 16-byte aligned");
  *a = pd::SelectArgs{};
  a->q_dec = q;
  a->key_mean = key_mean;
  a->tok_rank = tok_rank;
  a->chunk_score = chunk_score;
  a->chunk_idx = chunk_idx;
  a->tok_slot = tok_slot;
  a->B = d->batch;
  a->N = d->n_chunks;
  a->C = d->chunk_len;
  a->Hq = d->n_heads_q;
  a->Hkv = d->n_heads_kv;
  a->G = a->Hq / a->Hkv;
  a->Ld = d->dec_len;
  a->D = d->head_dim;
  a->K = top_k;
  a->Bt = tok_budget;
  a->q_rows = d->dec_len;
  a->q_row0 = 0;
  a->q_bstride = d->dec_len;
  a->NS = pd::select_row_splits(a->q_rows);
  a->bf16 = d->dtype == PD_BF16;
  a->scale = scale_of(d);
  return check_select_grid(d, a->q_rows);
}

void place_select_ws(void* ws, pd::SelectArgs* a) { a->partial = (float*)ws; }

}  // namespace

extern "C" {

pd_status pd_score_select(const pd_dims* d, int32_t top_k, int32_t tok_budget, const void* q_dec,
                          const float* key_mean, const int32_t* tok_rank, int32_t* chunk_idx, int32_t* tok_slot,
                          float* chunk_score, void* workspace, size_t ws_bytes, void* stream) {
  PD_RETURN_IF(check_dims(d));
  pd::SelectArgs a;
  PD_RETURN_IF(select_args(d, top_k, tok_budget, q_dec, key_mean, tok_rank, chunk_idx, tok_slot, chunk_score, &a));
  PD_RETURN_IF(check_ws(workspace, ws_bytes, select_ws(d)));
  place_select_ws(workspace, &a);
  return hip_status(pd::launch_score_select(a, (hipStream_t)stream), "score/select kernels");
}

pd_status pd_score_select_noalloc(const pd_dims* d, int32_t top_k, int32_t tok_budget, const void* q_dec,
                                  const float* key_mean, const int32_t* tok_rank, int32_t* chunk_idx,
                                  int32_t* tok_slot, float* chunk_score, void* stream) {
  PD_RETURN_IF(check_dims(d));
  pd::SelectArgs a;
  PD_RETURN_IF(select_args(d, top_k, tok_budget, q_dec, key_mean, tok_rank, chunk_idx, tok_slot, chunk_score, &a));
  const size_t need = select_ws(d);
  if (need > kNoallocScratchBytes)
    return fail(PD_ERR_BAD_DIMS,
                "selection needs %zu bytes of scratch (B*N*H_q*ceil(L_d/128)*4); the static scratch holds %zu",
                need, kNoallocScratchBytes);
  void* ws = nullptr;
  PD_RETURN_IF(scratch_of_current_device(&ws));
  place_select_ws(ws, &a);
  return hip_status(pd::launch_score_select(a, (hipStream_t)stream), "score/select kernels");
}

pd_status pd_score_select_static(const pd_dims* d, int32_t top_k, int32_t tok_budget, const void* q_qm,
                                 const float* key_mean, const int32_t* tok_rank, int32_t* chunk_idx,
                                 int32_t* tok_slot, float* chunk_score, void* workspace, size_t ws_bytes,
                                 void* stream) {
  PD_RETURN_IF(check_dims(d));
  if (d->m_len < 1) return fail(PD_ERR_BAD_DIMS, "m_len=%d: static selection needs pseudo-label rows", d->m_len);
  pd::SelectArgs a;
  PD_RETURN_IF(select_args(d, top_k, tok_budget, q_qm, key_mean, tok_rank, chunk_idx, tok_slot, chunk_score, &a));
  PD_RETURN_IF(check_ws(workspace, ws_bytes, select_ws(d)));
  place_select_ws(workspace, &a);
  // The L_m pseudo-label rows follow the L_q query rows of each sequence's q/m
  // block (chunk 0's copy when the rows are given per chunk).
  a.q_rows = d->m_len;
  a.q_row0 = d->q_len;
  a.q_bstride = (d->qm_per_chunk ? d->n_chunks : 1) * (d->q_len + d->m_len);
  a.NS = pd::select_row_splits(a.q_rows);
  PD_RETURN_IF(check_select_grid(d, a.q_rows));
  return hip_status(pd::launch_score_select(a, (hipStream_t)stream), "static score/select kernels");
}

pd_status pd_gather_selected(const pd_dims* d, int32_t top_k, int32_t tok_budget, const void* k_cache,
                             const void* v_cache, const int32_t* chunk_idx, const int32_t* tok_slot, void* k_sel,
                             void* v_sel, void* stream) {
  PD_RETURN_IF(check_dims(d));
  if (top_k < 1 || top_k > d->n_chunks)
    return fail(PD_ERR_BAD_DIMS, "top_k=%d must be in 1..n_chunks=%d", top_k, d->n_chunks);
  if (tok_budget < 1 || tok_budget > d->chunk_len)
    return fail(PD_ERR_BAD_DIMS, "tok_budget=%d must be in 1..chunk_len=%d", tok_budget, d->chunk_len);
  PD_REQUIRE_PTR(k_cache);
  PD_REQUIRE_PTR(v_cache);
  PD_REQUIRE_PTR(chunk_idx);
  PD_REQUIRE_PTR(tok_slot);
  PD_REQUIRE_PTR(k_sel);
  PD_REQUIRE_PTR(v_sel);
  if ((long long)d->batch * d->n_heads_kv * n_sel_of(top_k, tok_budget) * d->head_dim * elem_bytes(d) / 16 >=
      (1LL << 40))
    return fail(PD_ERR_BAD_DIMS, "compact buffer too large");
  return hip_status(pd::launch_gather_selected(k_cache, v_cache, chunk_idx, tok_slot, k_sel, v_sel, d->batch,
                                               d->n_chunks, d->chunk_len, d->n_heads_kv, top_k, tok_budget,
                                               d->head_dim * elem_bytes(d), (hipStream_t)stream),
                    "gather kernel");
}

pd_status pd_gather_joint(const pd_dims* d, int32_t top_k, int32_t tok_budget, const int32_t* chunk_idx,
                          const int32_t* tok_slot, const void* q_pre, const void* k_cache, const void* v_cache,
                          const void* q_qm, const void* k_qm, const void* v_qm, double rope_base, void* q_joint,
                          void* k_joint, void* v_joint, void* k_pref, void* v_pref, void* stream) {
  PD_RETURN_IF(check_dims(d));
  if (top_k < 1 || top_k > d->n_chunks)
    return fail(PD_ERR_BAD_DIMS, "top_k=%d must be in 1..n_chunks=%d", top_k, d->n_chunks);
  if (tok_budget < 1 || tok_budget > d->chunk_len)
    return fail(PD_ERR_BAD_DIMS, "tok_budget=%d must be in 1..chunk_len=%d", tok_budget, d->chunk_len);
  if (!std::isfinite(rope_base) || rope_base < 0.0)
    return fail(PD_ERR_BAD_DIMS, "rope_base must be finite and >= 0 (0: no rotation)");
  PD_REQUIRE_PTR(chunk_idx);
  PD_REQUIRE_PTR(tok_slot);
  PD_REQUIRE_PTR(q_pre);
  PD_REQUIRE_PTR(k_cache);
  PD_REQUIRE_PTR(v_cache);
  PD_REQUIRE_PTR(q_qm);
  PD_REQUIRE_PTR(k_qm);
  PD_REQUIRE_PTR(v_qm);
  PD_REQUIRE_PTR(q_joint);
  PD_REQUIRE_PTR(k_joint);
  PD_REQUIRE_PTR(v_joint);
  if ((k_pref == nullptr) != (v_pref == nullptr))
    return fail(PD_ERR_NULL_PTR, "k_pref and v_pref must be both given or both NULL");
  if (k_pref && (!aligned16(k_pref) || !aligned16(v_pref)))
    return fail(PD_ERR_MISALIGNED, "pointer 'k_pref' or 'v_pref' is not 16-byte aligned");
  const long long lj = n_sel_of(top_k, tok_budget) + d->q_len;
  if (lj * d->n_heads_q * d->head_dim >= (1LL << 31))
    return fail(PD_ERR_BAD_DIMS, "joint rows of one sequence (L_j*n_heads_q*head_dim) must stay below 2^31 elements");
  if ((long long)d->batch * lj >= (1LL << 31)) return fail(PD_ERR_BAD_DIMS, "batch*L_j must stay below 2^31");
  pd::JointArgs a{};
  a.q_pre = q_pre;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.q_qm = q_qm;
  a.k_qm = k_qm;
  a.v_qm = v_qm;
  a.chunk_idx = chunk_idx;
  a.tok_slot = tok_slot;
  a.q_joint = q_joint;
  a.k_joint = k_joint;
  a.v_joint = v_joint;
  a.k_pref = k_pref;
  a.v_pref = v_pref;
  a.B = d->batch;
  a.N = d->n_chunks;
  a.C = d->chunk_len;
  a.Lq = d->q_len;
  a.Lm = d->m_len;
  a.Hq = d->n_heads_q;
  a.Hkv = d->n_heads_kv;
  a.G = a.Hq / a.Hkv;
  a.D = d->head_dim;
  a.K = top_k;
  a.Bt = tok_budget;
  a.Lj = (int)lj;
  a.qm_per_chunk = d->qm_per_chunk;
  a.elem_bytes = elem_bytes(d);
  a.rope_base = rope_base;
  return hip_status(pd::launch_gather_joint(a, (hipStream_t)stream), "joint gather kernel");
}

// Shared by the gathered and the compact decode entry points (arguments checked
// by the caller except the common ones below).
static pd_status decode_core(const pd_dims* d, int top_k, int tok_budget, long long n_sel, bool compact,
                             const void* q_dec, const void* k_dec, const void* v_dec, const void* k_pref,
                             const void* v_pref, const int32_t* chunk_idx, const int32_t* tok_slot,
                             const void* k_static, const void* v_static, int32_t n_static, void* o_dec,
                             float* lse_dec, int32_t num_splits, void* workspace, size_t ws_bytes, void* stream) {
  if (n_static < 0 || n_static > d->q_len + d->m_len)
    return fail(PD_ERR_BAD_DIMS, "n_static=%d must be in 0..q_len+m_len=%d", n_static, d->q_len + d->m_len);
  if (num_splits < 0 || num_splits > kMaxSplits)
    return fail(PD_ERR_BAD_DIMS, "num_splits=%d must be in 0..%d", num_splits, kMaxSplits);
  PD_REQUIRE_PTR(q_dec);
  PD_REQUIRE_PTR(k_dec);
  PD_REQUIRE_PTR(v_dec);
  PD_REQUIRE_PTR(o_dec);
  if (n_static > 0) {
    PD_REQUIRE_PTR(k_static);
    PD_REQUIRE_PTR(v_static);
  }
  if (lse_dec && !aligned16(lse_dec)) return fail(PD_ERR_MISALIGNED, "pointer 'lse_dec' is not 16-byte aligned");
  PD_RETURN_IF(check_decode_rows(d, n_sel, n_static));
  const int S_req = requested_splits(d, n_sel, num_splits);
  const int S = effective_splits(d, n_sel, n_static, num_splits);
  PD_RETURN_IF(check_decode_grid(d, S_req));
  PD_RETURN_IF(check_ws(workspace, ws_bytes, decode_ws_bytes(d, S_req)));

  const bool bf16 = d->dtype == PD_BF16;
  hipStream_t s = (hipStream_t)stream;
  pd::DecodeArgs a{};
  a.q_dec = (const uint16_t*)q_dec;
  a.k_dec = (const uint16_t*)k_dec;
  a.v_dec = (const uint16_t*)v_dec;
  a.k_cache = (const uint16_t*)k_pref;
  a.v_cache = (const uint16_t*)v_pref;
  a.k_static = (const uint16_t*)k_static;
  a.v_static = (const uint16_t*)v_static;
  a.chunk_idx = chunk_idx;
  a.tok_slot = tok_slot;
  a.o_dec = o_dec;
  a.lse_dec = lse_dec;
  a.B = d->batch;
  a.N = d->n_chunks;
  a.C = d->chunk_len;
  a.Hq = d->n_heads_q;
  a.Hkv = d->n_heads_kv;
  a.G = a.Hq / a.Hkv;
  a.Ld = d->dec_len;
  a.Ls = d->q_len + d->m_len;
  a.K = top_k;
  a.Bt = tok_budget;
  a.n_sel = (int)n_sel;
  a.compact = compact ? 1 : 0;
  a.n_static = n_static;
  a.S = S;
  a.out_f32 = d->out_fp32;
  a.scale_log2 = scale_of(d) * 1.4426950408889634f;
  a.n_qt = decode_qtiles(d);
  a.total = (int)(decode_units(d) * S);
  if (S > 1) {
    const size_t rows = (size_t)S * a.B * a.Hq * a.Ld;
    a.o_part = (float*)workspace;
    a.lse_part = (float*)((char*)workspace + round_up(rows * d->head_dim * sizeof(float)));
  }
  hipError_t err = bf16 ? pd::launch_decode_bf16(a, d->head_dim, s) : pd::launch_decode_f32(a, d->head_dim, s);
  if (err != hipSuccess) return hip_status(err, "decode kernel");
  if (S > 1) {
    err = pd::launch_merge(a.o_part, a.lse_part, o_dec, lse_dec, S, a.B, a.Hq, a.Ld, d->head_dim,
                           bf16 && !d->out_fp32, s);
    if (err != hipSuccess) return hip_status(err, "merge kernel");
  }
  return PD_OK;
}

pd_status pd_sparse_decode_attn(const pd_dims* d, int32_t top_k, int32_t tok_budget, const void* q_dec,
                                const void* k_dec, const void* v_dec, const void* k_cache, const void* v_cache,
                                const int32_t* chunk_idx, const int32_t* tok_slot, const void* k_static,
                                const void* v_static, int32_t n_static, void* o_dec, float* lse_dec,
                                int32_t num_splits, void* workspace, size_t ws_bytes, void* stream) {
  PD_RETURN_IF(check_dims(d));
  if (top_k < 1 || top_k > d->n_chunks)
    return fail(PD_ERR_BAD_DIMS, "top_k=%d must be in 1..n_chunks=%d", top_k, d->n_chunks);
  if (tok_budget < 1 || tok_budget > d->chunk_len)
    return fail(PD_ERR_BAD_DIMS, "tok_budget=%d must be in 1..chunk_len=%d", tok_budget, d->chunk_len);
  PD_REQUIRE_PTR(k_cache);
  PD_REQUIRE_PTR(v_cache);
  PD_REQUIRE_PTR(chunk_idx);
  PD_REQUIRE_PTR(tok_slot);
  return decode_core(d, top_k, tok_budget, n_sel_of(top_k, tok_budget), false, q_dec, k_dec, v_dec, k_cache,
                     v_cache, chunk_idx, tok_slot, k_static, v_static, n_static, o_dec, lse_dec, num_splits,
                     workspace, ws_bytes, stream);
}

pd_status pd_sparse_decode_attn_compact(const pd_dims* d, int32_t n_sel, const void* q_dec, const void* k_dec,
                                        const void* v_dec, const void* k_sel, const void* v_sel,
                                        const void* k_static, const void* v_static, int32_t n_static, void* o_dec,
                                        float* lse_dec, int32_t num_splits, void* workspace, size_t ws_bytes,
                                        void* stream) {
  PD_RETURN_IF(check_dims(d));
  if (n_sel < 0 || n_sel > kMaxCompactRows)
    return fail(PD_ERR_BAD_DIMS, "n_sel=%d must be in 0..%d", n_sel, kMaxCompactRows);
  if (n_sel > 0) {
    PD_REQUIRE_PTR(k_sel);
    PD_REQUIRE_PTR(v_sel);
  }
  return decode_core(d, 0, 0, n_sel, true, q_dec, k_dec, v_dec, k_sel, v_sel, nullptr, nullptr, k_static,
                     v_static, n_static, o_dec, lse_dec, num_splits, workspace, ws_bytes, stream);
}

size_t pd_compact_workspace_bytes(const pd_dims* d, int32_t n_sel, int32_t num_splits) {
  if (check_dims(d) != PD_OK || n_sel < 0 || n_sel > kMaxCompactRows || num_splits < 0 || num_splits > kMaxSplits)
    return 0;
  if (check_decode_rows(d, n_sel, 0) != PD_OK) return 0;
  const int S = requested_splits(d, n_sel, num_splits);
  if (check_decode_grid(d, S) != PD_OK) return 0;
  return decode_ws_bytes(d, S);
}

}  // extern "C"
