// Host-side argument validation of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer: every entry point is called with arguments it
// must reject before launching anything (so no GPU is needed), plus the size
// queries and status strings.  Exit status 0 iff every call returned the
// expected status; the sanitizers abort on any memory or UB error.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "pd.h"

static int failures = 0;

#define EXPECT(call, want)                                                                     \
  do {                                                                                         \
    const pd_status got_ = (call);                                                             \
    if (got_ != (want)) {                                                                      \
      std::printf("FAIL line %d: %s -> %d (want %d): %s\n", __LINE__, #call, (int)got_, (int)(want), \
                  pd_last_error_message());                                                    \
      ++failures;                                                                              \
    }                                                                                          \
  } while (0)

static pd_dims dims() {
  pd_dims d;
  std::memset(&d, 0, sizeof(d));
  d.batch = 1; d.n_chunks = 4; d.chunk_len = 128; d.q_len = 16; d.m_len = 32; d.dec_len = 32;
  d.n_heads_q = 4; d.n_heads_kv = 4; d.head_dim = 64; d.dtype = PD_BF16;
  return d;
}

int main() {
  void* A = reinterpret_cast<void*>(uintptr_t(1) << 20);        // fake aligned device address
  void* MIS = reinterpret_cast<void*>((uintptr_t(1) << 20) + 8);  // misaligned
  float* Af = static_cast<float*>(A);
  int32_t* Ai = static_cast<int32_t*>(A);
  const size_t big = size_t(1) << 30;

  // dims checks (through the prefill)
  pd_dims d = dims();
  EXPECT(pd_prefill_chunks(nullptr, A, A, A, A, A, A, A, A, A, Af, Ai, Af, nullptr, A, big, nullptr), PD_ERR_NULL_PTR);
  const struct { int32_t pd_dims::*f; int32_t v; pd_status want; } bad[] = {
      {&pd_dims::batch, 0, PD_ERR_BAD_DIMS},      {&pd_dims::n_chunks, 1025, PD_ERR_BAD_DIMS},
      {&pd_dims::chunk_len, 0, PD_ERR_BAD_DIMS},  {&pd_dims::chunk_len, 5000, PD_ERR_BAD_DIMS},
      {&pd_dims::q_len, 0, PD_ERR_BAD_DIMS},      {&pd_dims::m_len, -1, PD_ERR_BAD_DIMS},
      {&pd_dims::dec_len, 0, PD_ERR_BAD_DIMS},    {&pd_dims::n_heads_kv, 3, PD_ERR_UNSUPPORTED},
      {&pd_dims::head_dim, 96, PD_ERR_UNSUPPORTED}, {&pd_dims::dtype, 7, PD_ERR_UNSUPPORTED},
      {&pd_dims::qm_per_chunk, 2, PD_ERR_BAD_DIMS}, {&pd_dims::out_fp32, -1, PD_ERR_BAD_DIMS},
      {&pd_dims::tok_score_dir, 5, PD_ERR_BAD_DIMS},
  };
  for (const auto& b : bad) {
    pd_dims x = dims();
    x.*(b.f) = b.v;
    EXPECT(pd_prefill_chunks(&x, A, A, A, A, A, A, A, A, A, Af, Ai, Af, nullptr, A, big, nullptr), b.want);
    if (pd_workspace_bytes(&x, 2, 64, 0, 0) != 0) { std::printf("FAIL: size query accepted bad dims\n"); ++failures; }
  }
  pd_dims huge = dims();
  huge.n_chunks = 1024; huge.chunk_len = 4096; huge.n_heads_kv = 64; huge.n_heads_q = 64; huge.head_dim = 128;
  EXPECT(pd_prefill_chunks(&huge, A, A, A, A, A, A, A, A, A, Af, Ai, Af, nullptr, A, big, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_prefill_chunks(&d, nullptr, A, A, A, A, A, A, A, A, Af, Ai, Af, nullptr, A, big, nullptr), PD_ERR_NULL_PTR);
  EXPECT(pd_prefill_chunks(&d, A, A, A, A, A, A, MIS, A, A, Af, Ai, Af, nullptr, A, big, nullptr), PD_ERR_MISALIGNED);
  EXPECT(pd_prefill_chunks(&d, A, A, A, A, A, A, A, A, A, Af, Ai, Af, nullptr, nullptr, big, nullptr), PD_ERR_WORKSPACE);
  EXPECT(pd_prefill_chunks(&d, A, A, A, A, A, A, A, A, A, Af, Ai, Af, nullptr, A, 16, nullptr), PD_ERR_WORKSPACE);

  // selection
  const size_t ws1 = pd_workspace_bytes(&d, 2, 64, 0, 1);
  EXPECT(pd_score_select(&d, 0, 64, A, Af, Ai, Ai, Ai, nullptr, A, ws1, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_score_select(&d, 5, 64, A, Af, Ai, Ai, Ai, nullptr, A, ws1, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_score_select(&d, 2, 129, A, Af, Ai, Ai, Ai, nullptr, A, ws1, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_score_select(&d, 2, 64, nullptr, Af, Ai, Ai, Ai, nullptr, A, ws1, nullptr), PD_ERR_NULL_PTR);
  EXPECT(pd_score_select(&d, 2, 64, A, Af, Ai, Ai, Ai, static_cast<float*>(MIS), A, ws1, nullptr), PD_ERR_MISALIGNED);
  EXPECT(pd_score_select(&d, 2, 64, A, Af, Ai, Ai, Ai, nullptr, A, ws1 - 1, nullptr), PD_ERR_WORKSPACE);
  EXPECT(pd_score_select_static(&d, 2, 64, nullptr, Af, Ai, Ai, Ai, nullptr, A, ws1, nullptr), PD_ERR_NULL_PTR);
  EXPECT(pd_score_select_noalloc(&d, 0, 64, A, Af, Ai, Ai, Ai, nullptr, nullptr), PD_ERR_BAD_DIMS);
  pd_dims over = dims();
  over.batch = 64; over.n_chunks = 1024; over.chunk_len = 64; over.n_heads_q = 64; over.n_heads_kv = 8;
  over.dec_len = 512; over.head_dim = 128;
  EXPECT(pd_score_select_noalloc(&over, 4, 8, A, Af, Ai, Ai, Ai, nullptr, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_select_ranked(&d, 2, 64, Af, 2, Ai, Ai, Ai, nullptr), PD_ERR_BAD_DIMS);

  // decode
  EXPECT(pd_sparse_decode_attn(&d, 2, 64, A, A, A, A, A, Ai, Ai, A, A, 49, A, nullptr, 0, A, big, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_sparse_decode_attn(&d, 2, 64, A, A, A, A, A, Ai, Ai, nullptr, nullptr, 16, A, nullptr, 0, A, big, nullptr), PD_ERR_NULL_PTR);
  EXPECT(pd_sparse_decode_attn(&d, 2, 64, A, A, A, A, A, Ai, Ai, A, A, 16, A, nullptr, 65, A, big, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_sparse_decode_attn(&d, 2, 64, A, A, A, A, A, Ai, Ai, A, A, 16, A, static_cast<float*>(MIS), 1, A, big, nullptr), PD_ERR_MISALIGNED);
  const size_t ws2 = pd_workspace_bytes(&d, 2, 64, 4, 2);
  EXPECT(pd_sparse_decode_attn(&d, 2, 64, A, A, A, A, A, Ai, Ai, A, A, 16, A, nullptr, 4, A, ws2 - 1, nullptr), PD_ERR_WORKSPACE);
  pd_dims wide = dims();
  wide.n_heads_q = 32; wide.n_heads_kv = 32; wide.head_dim = 128;
  EXPECT(pd_sparse_decode_attn_compact(&wide, 1 << 20, A, A, A, A, A, A, A, 16, A, nullptr, 0, A, big, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_sparse_decode_attn_compact(&d, -1, A, A, A, A, A, A, A, 16, A, nullptr, 0, A, big, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_gather_selected(&d, 5, 64, A, A, Ai, Ai, A, A, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_gather_joint(&d, 2, 64, Ai, Ai, A, A, A, A, A, A, -1.0, A, A, A, nullptr, nullptr, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_gather_joint(&d, 2, 64, Ai, Ai, A, A, A, A, A, A, 1e4, A, A, A, A, nullptr, nullptr), PD_ERR_NULL_PTR);
  EXPECT(pd_mfma_rate_probe(0, 10, Af, nullptr), PD_ERR_BAD_DIMS);
  // launch grids past one dimension: decode work items and chunk-score splits
  pd_dims tall = dims();
  tall.batch = 1 << 20; tall.n_chunks = 1; tall.chunk_len = 1; tall.q_len = 1; tall.m_len = 0;
  tall.dec_len = 1 << 19; tall.n_heads_q = 1; tall.n_heads_kv = 1; tall.head_dim = 128;
  EXPECT(pd_score_select(&tall, 1, 1, A, Af, Ai, Ai, Ai, nullptr, A, big, nullptr), PD_ERR_BAD_DIMS);
  EXPECT(pd_sparse_decode_attn(&tall, 1, 1, A, A, A, A, A, Ai, Ai, A, A, 1, A, nullptr, 0, A, big, nullptr), PD_ERR_BAD_DIMS);
  if (pd_workspace_bytes(&tall, 1, 1, 0, 2) != 0) { std::printf("FAIL: size query accepted a huge decode\n"); ++failures; }

  // queries and strings
  if (pd_cache_bytes(&d) != size_t(1) * 4 * 4 * 129 * 64 * 2) { std::printf("FAIL: pd_cache_bytes\n"); ++failures; }
  if (pd_decode_splits(&d, 2, 64, 16, 3) != 3) { std::printf("FAIL: pd_decode_splits\n"); ++failures; }
  for (int s = 0; s <= 7; ++s)
    if (!pd_status_string(static_cast<pd_status>(s)) || !*pd_status_string(static_cast<pd_status>(s))) ++failures;
  if (!std::strstr(pd_version(), "gfx950")) ++failures;
  std::printf("%s (%d failures)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
