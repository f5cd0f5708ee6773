// Stage (b): per-step chunk scores, top-K chunks and the kept tokens of each
// kept chunk, plus the once-per-layer token ranking of stage (a).
//
//   token_rank: grid (b, n)     -- bitonic sort of the C Eq. 5 scores in LDS
//                                  (score desc, index asc) -> rank of each token;
//   qscore:     grid (b, h, sp) -- by linearity the chunk score splits into
//                                  terms scale * <(1/L_d) sum_{r in sp} q_r, kbar_n>
//                                  over heads and row splits: one workgroup sums
//                                  its rows of one head, then dots with all N
//                                  key means of that head's KV group;
//   gather:     grid (rows)     -- static-selection mode: kept rows copied once
//                                  into a contiguous per-(sequence, KV head) buffer;
//   chunk_score: grid (b, n)    -- prefill-time chunk score from the content
//                                  mass of the query and pseudo-label rows;
//   select:     grid (b, k)     -- sums the terms of every chunk in a fixed
//                                  order, ranks the N scores (bitonic sort in
//                                  LDS), takes the k-th kept chunk in ascending
//                                  order and writes its tokens with rank < B_tok
//                                  in ascending slot order (flags + block scan).
// All reductions run in a fixed order, so results are bitwise reproducible.
#include "pd_common.h"
#include "pd_kernels.h"

namespace pd {

// 16 bytes of elements as floats: 8 bf16 or 4 fp32.
template <bool BF16>
struct Vec16 {
  static constexpr int E = BF16 ? 8 : 4;
  __device__ static void load(const void* base, size_t elem_off, float (&v)[E]) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(
        reinterpret_cast<const char*>(base) + elem_off * (BF16 ? 2 : 4));
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(w[i]);
    }
  }
};

// Sum of `nrows` rows (stride `row_stride` elements) of D elements each,
// starting at element `base_off`; returns the D sums * `mul` into out[0..D).
// 256 threads: thread t reads 16-byte chunk (t % TPR) of rows t/TPR, +NG, ...
template <bool BF16>
__device__ void rows_mean(const void* src, size_t base_off, size_t row_stride, int nrows, int D,
                          float mul, float* out, float* red /* [256/TPR][D] */) {
  constexpr int E = Vec16<BF16>::E;
  const int TPR = D / E, NG = 256 / TPR;
  const int t = threadIdx.x, c = t % TPR, rg = t / TPR;
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  for (int r = rg; r < nrows; r += NG) {
    float v[E];
    Vec16<BF16>::load(src, base_off + (size_t)r * row_stride + c * E, v);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += v[e];
  }
#pragma unroll
  for (int e = 0; e < E; ++e) red[rg * D + c * E + e] = acc[e];
  __syncthreads();
  if (t < D) {
    float s = 0.f;
    for (int g = 0; g < NG; ++g) s += red[g * D + t];
    out[t] = s * mul;
  }
}

template <bool BF16>
__global__ __launch_bounds__(256) void key_mean_kernel(const void* k_cache, float* key_mean, int C, int D) {
  __shared__ float red[2048];
  const size_t bng = blockIdx.x;  // ((b*N + n)*Hkv + g)
  rows_mean<BF16>(k_cache, (bng * (C + 1) + 1) * D, (size_t)D, C, D, 1.0f / C, key_mean + bng * D, red);
}

__device__ __forceinline__ uint64_t rank_key(float score, int idx) {
  return ((uint64_t)(~float_order_key(score)) << 32) | (uint32_t)idx;
}

// Ascending bitonic sort of P (power of two) keys in LDS, 256 threads.
__device__ void bitonic_sort(uint64_t* keys, int P) {
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < P; i += 256) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = keys[i], c = keys[ixj];
          const bool up = (i & k) == 0;
          if ((a > c) == up) {
            keys[i] = c;
            keys[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

static int next_pow2(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Rank of every token of one chunk by its Eq. 5 score.
__global__ __launch_bounds__(256) void token_rank_kernel(const float* tok_score, int32_t* tok_rank, int C,
                                                          int Cpad) {
  extern __shared__ __attribute__((aligned(16))) uint64_t keys[];
  const size_t bn = blockIdx.x;
  const float* e = tok_score + bn * C;
  for (int j = threadIdx.x; j < Cpad; j += 256) keys[j] = j < C ? rank_key(e[j], j) : ~0ull;
  __syncthreads();
  bitonic_sort(keys, Cpad);
  for (int i = threadIdx.x; i < C; i += 256) tok_rank[bn * C + (uint32_t)keys[i]] = i;
}

// Ascending bitonic sort of P (power of two) keys in LDS by NT threads.
template <int NT>
__device__ void bitonic_sort_nt(uint64_t* keys, int P) {
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < P; i += NT) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = keys[i], c = keys[ixj];
          const bool up = (i & k) == 0;
          if ((a > c) == up) {
            keys[i] = c;
            keys[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

// Workgroups (b*N + n, 0): e of one chunk = sum over the H_q heads of the
// per-head sums (heads in ascending order), written out, then every token's
// rank as token_rank_kernel, with 1024 threads (one compare per thread per
// sort stage at C = 1024).  Workgroups (b*N + n, y >= 1): the chunk's key means
// k-bar[g][d] = (1/C) * the sum of the km_slots partial sums of the
// cache-writing workgroups (fixed order); these workgroups (at most 64 per
// chunk) take 1024 of the H_kv*d values at a time.
constexpr int kRankThreads = 1024;
__global__ __launch_bounds__(kRankThreads) void head_sum_rank_kernel(const float* per_head, float* tok_score,
                                                                      int32_t* tok_rank, int Hq, int C, int Cpad,
                                                                      const float* km_part, float* key_mean, int HD,
                                                                      int D, int km_slots) {
  extern __shared__ __attribute__((aligned(16))) uint64_t keys[];
  const size_t bn = blockIdx.x;
  if (blockIdx.y > 0) {
    for (int i = (blockIdx.y - 1) * kRankThreads + threadIdx.x; i < HD; i += (gridDim.y - 1) * kRankThreads) {
      const int g = i / D, d = i % D;
      const float* src = km_part + ((bn * (HD / D) + g) * (size_t)km_slots) * D + d;
      float sum = 0.f;
#pragma unroll 8
      for (int q = 0; q < km_slots; ++q) sum += src[(size_t)q * D];
      key_mean[bn * HD + i] = sum * (1.0f / C);
    }
    return;
  }
  const float* ph = per_head + bn * Hq * C;
  for (int j = threadIdx.x; j < Cpad; j += kRankThreads) {
    if (j < C) {
      float e = 0.f;
#pragma unroll 16
      for (int h = 0; h < Hq; ++h) e += ph[(size_t)h * C + j];
      tok_score[bn * C + j] = e;
      keys[j] = rank_key(e, j);
    } else {
      keys[j] = ~0ull;
    }
  }
  __syncthreads();
  bitonic_sort_nt<kRankThreads>(keys, Cpad);
  for (int i = threadIdx.x; i < C; i += kRankThreads) tok_rank[bn * C + (uint32_t)keys[i]] = i;
}

hipError_t launch_head_sum_rank(const float* per_head, float* tok_score, int32_t* tok_rank, int B, int N, int Hq,
                                int C, const float* km_part, float* key_mean, int Hkv, int D, int km_slots,
                                hipStream_t s) {
  const int Cpad = next_pow2(C);
  const int HD = Hkv * D;
  const dim3 grid(B * N, 1 + std::min(64, (HD + kRankThreads - 1) / kRankThreads));
  hipLaunchKernelGGL(head_sum_rank_kernel, grid, dim3(kRankThreads), (size_t)Cpad * 8, s, per_head, tok_score,
                     tok_rank, Hq, C, Cpad, km_part, key_mean, HD, D, km_slots);
  return hipGetLastError();
}

hipError_t launch_token_rank(const float* tok_score, int32_t* tok_rank, int B, int N, int C, hipStream_t s) {
  const int Cpad = next_pow2(C);
  hipLaunchKernelGGL(token_rank_kernel, dim3(B * N), dim3(256), (size_t)Cpad * 8, s, tok_score, tok_rank, C, Cpad);
  return hipGetLastError();
}

// Decode rows per score workgroup.
constexpr int kScoreRows = 128;
int select_row_splits(int Ld) { return (Ld + kScoreRows - 1) / kScoreRows; }

// Chunk-score terms of one (b, h, row split): scale * <(1/L_d) sum_r q_r, kbar[b][n][h/G]> for all n.
// Latency-bound (a few KB per workgroup), so every load of a thread is issued
// before the first use: the key means of the first 32 chunks, then the thread's
// share of the rows (fully unrolled).  The row sums are reduced through LDS in
// a fixed order; the dot products run 8 lanes per chunk (D/8 dimensions each),
// reduced by a fixed xor butterfly.  Workgroup id: heads fastest, then row
// split, then sequence.
template <bool BF16, int D>
__device__ __forceinline__ void qscore_terms(const SelectArgs& a, int bid) {
  constexpr int SL = D / 8;
  constexpr int E = Vec16<BF16>::E;
  constexpr int TPR = D / E, NG = 256 / TPR, IT = kScoreRows / NG;
  __shared__ float red[NG * D];
  __shared__ float qp[D];
  const int N = a.N, Hq = a.Hq, NS = a.NS;
  const int h = bid % Hq;
  const int sp = (bid / Hq) % NS;
  const int b = bid / (Hq * NS);
  const int t = threadIdx.x;
  const int r0 = sp * kScoreRows, nr = min(a.q_rows, r0 + kScoreRows) - r0;
  const float* kb = a.key_mean + ((size_t)b * N * a.Hkv + h / a.G) * D;
  const int j = t & 7;
  f32x4 kv[SL / 4];
  {
    const int n = t >> 3;
    if (n < N) {
      const f32x4* kr = reinterpret_cast<const f32x4*>(kb + (size_t)n * a.Hkv * D + j * SL);
#pragma unroll
      for (int i = 0; i < SL / 4; ++i) kv[i] = kr[i];
    }
  }
  const int c = t % TPR, rg = t / TPR;
  const size_t base = (((size_t)b * a.q_bstride + a.q_row0 + r0) * Hq + h) * D + c * E;
  u32x4 w[IT];
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    const int r = rg + it * NG;
    w[it] = r < nr ? *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(a.q_dec) +
                                                      (base + (size_t)r * Hq * D) * (BF16 ? 2 : 4))
                   : u32x4{0u, 0u, 0u, 0u};
  }
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll
  for (int it = 0; it < IT; ++it) {
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] += __uint_as_float(w[it][i] << 16);
        acc[2 * i + 1] += __uint_as_float(w[it][i] & 0xffff0000u);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[i] += __uint_as_float(w[it][i]);
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) red[rg * D + c * E + e] = acc[e];
  __syncthreads();
  if (t < D) {
    float sum = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) sum += red[g * D + t];
    qp[t] = sum * (1.0f / a.q_rows);
  }
  __syncthreads();
  float q[SL];
#pragma unroll
  for (int i = 0; i < SL; ++i) q[i] = qp[j * SL + i];
  for (int n0 = 0; n0 < N; n0 += 32) {
    const int n = n0 + (t >> 3);
    if (n0 > 0 && n < N) {
      const f32x4* kr = reinterpret_cast<const f32x4*>(kb + (size_t)n * a.Hkv * D + j * SL);
#pragma unroll
      for (int i = 0; i < SL / 4; ++i) kv[i] = kr[i];
    }
    float acc2 = 0.f;
    if (n < N) {
#pragma unroll
      for (int i = 0; i < SL / 4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc2 = fmaf(q[4 * i + e], kv[i][e], acc2);
    }
    acc2 += __shfl_xor(acc2, 1);
    acc2 += __shfl_xor(acc2, 2);
    acc2 += __shfl_xor(acc2, 4);
    if (j == 0 && n < N) a.partial[((size_t)b * N + n) * Hq * NS + (size_t)h * NS + sp] = acc2 * a.scale;
  }
}

template <bool BF16, int D>
__global__ __launch_bounds__(256) void qscore_kernel(SelectArgs a) {
  qscore_terms<BF16, D>(a, blockIdx.x);
}

// Chunk scores of sequence b: the T terms of each chunk summed 8 lanes per
// chunk (lane j sums terms j, j+8, ...), then a fixed xor butterfly over the 8
// lanes; keys[n] = rank key of the score (negated when neg), keys past N =
// max.  Writes chunk_score[b][n] when `out` is given.
__device__ void chunk_keys(const float* partial, int b, int N, int T, int Npad, int neg, uint64_t* keys,
                           float* out) {
  const int t = threadIdx.x;
  for (int n = t; n < Npad; n += 256) keys[n] = ~0ull;
  __syncthreads();
  const int j = t & 7;
  for (int n0 = 0; n0 < N; n0 += 32) {
    const int n = n0 + (t >> 3);
    float s = 0.f;
    if (n < N) {
      const float* pr = partial + ((size_t)b * N + n) * T;
#pragma unroll 16
      for (int i = j; i < T; i += 8) s += pr[i];
    }
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    if (j == 0 && n < N) {
      keys[n] = rank_key(neg ? -s : s, n);
      if (out) out[(size_t)b * N + n] = s;
    }
  }
  __syncthreads();
}

// Kept tokens (rank < Bt) of one chunk in ascending order: counts over
// contiguous segments, an exclusive scan (within each wave by shuffles, then
// across the 4 waves), then each segment writes its slots (token + 1).  The
// ranks of a segment are loaded 16 at a time, all in flight before the first
// compare (a plain loop waits for each load in turn).
__device__ void list_tokens(const int32_t* rk, int C, int Bt, int32_t* out, int* wsum) {
  constexpr int U = 16;
  const int t = threadIdx.x;
  const int seg = (C + 255) / 256;
  const int j0 = min(C, t * seg), j1 = min(C, j0 + seg);
  int cnt = 0;
  for (int base = j0; base < j1; base += U) {
    int r[U];
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = base + u < j1 ? rk[base + u] : Bt;
#pragma unroll
    for (int u = 0; u < U; ++u) cnt += r[u] < Bt;
  }
  const int lane = t & 63, wv = t >> 6;
  int inc = cnt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o);
    if (lane >= o) inc += y;
  }
  if (lane == 63) wsum[wv] = inc;
  __syncthreads();
  int pos = inc - cnt;
  for (int w = 0; w < wv; ++w) pos += wsum[w];
  for (int base = j0; base < j1; base += U) {
    int r[U];
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = base + u < j1 ? rk[base + u] : Bt;
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (r[u] < Bt) out[pos++] = base + u + 1;
  }
}

// neg = 1 keeps the K lowest scores instead of the K highest.  One workgroup
// per (sequence, kept chunk k): all compute the chunk ranking, workgroup k then
// lists the kept tokens of the k-th kept chunk.
__global__ __launch_bounds__(256) void select_kernel(const float* partial, const int32_t* tok_rank,
                                                      float* chunk_score, int32_t* chunk_idx, int32_t* tok_slot,
                                                      int N, int C, int K, int Bt, int T, int Npad, int neg) {
  extern __shared__ __attribute__((aligned(16))) uint64_t keys[];
  __shared__ int rankv[256];
  __shared__ int wsum[4];
  __shared__ int my_chunk;
  const int b = blockIdx.x / K, k = blockIdx.x % K;
  const int t = threadIdx.x;
  chunk_keys(partial, b, N, T, Npad, neg, keys, k == 0 ? chunk_score : nullptr);
  if (N <= 256) {
    if (t < N) {
      const uint64_t me = keys[t];
      int r = 0;
      for (int i = 0; i < N; ++i) r += keys[i] < me;
      rankv[t] = r;
    }
    __syncthreads();
    if (t < N && rankv[t] < K) {
      int pos = 0;
      for (int i = 0; i < t; ++i) pos += rankv[i] < K;
      if (pos == k) my_chunk = t;
      if (k == 0) chunk_idx[(size_t)b * K + pos] = t;
    }
  } else {
    bitonic_sort(keys, Npad);
    for (int i = t; i < K; i += 256) {
      const int x = (int)(uint32_t)keys[i];
      int pos = 0;
      for (int j = 0; j < K; ++j) pos += (int)(uint32_t)keys[j] < x;
      if (pos == k) my_chunk = x;
      if (k == 0) chunk_idx[(size_t)b * K + pos] = x;
    }
  }
  __syncthreads();
  list_tokens(tok_rank + ((size_t)b * N + my_chunk) * C, C, Bt, tok_slot + ((size_t)b * K + k) * Bt, wsum);
}

hipError_t launch_score_select(const SelectArgs& a, hipStream_t s) {
  const dim3 g1(a.B * a.Hq * a.NS);
  const int Npad = next_pow2(a.N);
#define PD_QSCORE(BF, DD) hipLaunchKernelGGL((qscore_kernel<BF, DD>), g1, dim3(256), 0, s, a)
  if (a.D == 128) {
    if (a.bf16) PD_QSCORE(true, 128); else PD_QSCORE(false, 128);
  } else {
    if (a.bf16) PD_QSCORE(true, 64); else PD_QSCORE(false, 64);
  }
#undef PD_QSCORE
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(select_kernel, dim3(a.B * a.K), dim3(256), (size_t)Npad * 8, s, a.partial, a.tok_rank,
                     a.chunk_score, a.chunk_idx, a.tok_slot, a.N, a.C, a.K, a.Bt, a.Hq * a.NS, Npad, 0);
  return hipGetLastError();
}

// Selection from scores the caller supplies (one term per chunk).
hipError_t launch_select_ranked(const float* chunk_score, int lowest, const int32_t* tok_rank, int32_t* chunk_idx,
                                int32_t* tok_slot, int B, int N, int C, int K, int Bt, hipStream_t s) {
  const int Npad = next_pow2(N);
  hipLaunchKernelGGL(select_kernel, dim3(B * K), dim3(256), (size_t)Npad * 8, s, chunk_score, tok_rank,
                     (float*)nullptr, chunk_idx, tok_slot, N, C, K, Bt, 1, Npad, lowest);
  return hipGetLastError();
}

// Prefill-time chunk score of one (b, n) from the per-head content masses of
// its L_q + L_m query and pseudo-label rows: a(r) = (1/H_q) sum_h mass[h][r],
// s = -(1/L_q) sum_{r < L_q} ln a(r) - (1/L_m) sum_{r >= L_q} ln a(r) (the
// second term only when L_m > 0).  Thread t takes rows t, t + 256, ...; both
// sums are reduced by a fixed tree, so the result is reproducible.
__global__ __launch_bounds__(256) void chunk_score_kernel(const float* qm_mass, float* chunk_score, int Hq, int Lq,
                                                           int Lm) {
  __shared__ float red[2][256];
  const size_t bn = blockIdx.x;
  const int R = Lq + Lm, t = threadIdx.x;
  const float* m = qm_mass + bn * Hq * R;
  float si = 0.f, sp = 0.f;
  for (int r = t; r < R; r += 256) {
    float a = 0.f;
    for (int h = 0; h < Hq; ++h) a += m[(size_t)h * R + r];
    const float nl = -logf(a / Hq);
    if (r < Lq) si += nl;
    else sp += nl;
  }
  red[0][t] = si;
  red[1][t] = sp;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) {
      red[0][t] += red[0][t + w];
      red[1][t] += red[1][t + w];
    }
    __syncthreads();
  }
  if (t == 0) chunk_score[bn] = red[0][0] / Lq + (Lm > 0 ? red[1][0] / Lm : 0.f);
}

hipError_t launch_chunk_score(const float* qm_mass, float* chunk_score, int B, int N, int Hq, int Lq, int Lm,
                              hipStream_t s) {
  hipLaunchKernelGGL(chunk_score_kernel, dim3(B * N), dim3(256), 0, s, qm_mass, chunk_score, Hq, Lq, Lm);
  return hipGetLastError();
}

// Static-selection mode: copy the kept rows of every (sequence, KV head) into a
// contiguous buffer [B][Hkv][K*(1+Bt)][row]: per kept chunk (ascending), its BOS
// row (slot 0) and then its kept slots.  16 bytes per thread.
__global__ __launch_bounds__(256) void gather_selected_kernel(const u32x4* k_cache, const u32x4* v_cache,
                                                               const int32_t* chunk_idx, const int32_t* tok_slot,
                                                               u32x4* k_sel, u32x4* v_sel, size_t total, int N,
                                                               int C1, int Hkv, int K, int Bt, int cpr) {
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= total) return;
  const int n_sel = K * (1 + Bt);
  const int c = (int)(gid % cpr);
  size_t r = gid / cpr;
  const int j = (int)(r % n_sel);
  r /= n_sel;
  const int g = (int)(r % Hkv);
  const int b = (int)(r / Hkv);
  const int kk = j / (1 + Bt), sl = j - kk * (1 + Bt);
  int slot = sl == 0 ? 0 : tok_slot[((size_t)b * K + kk) * Bt + sl - 1];
  int chunk = chunk_idx[(size_t)b * K + kk];
  const bool bad = kCheckIndices && !kept_row_ok(chunk, slot, sl == 0, N, C1 - 1);
  if (bad) chunk = slot = 0;
  const size_t src = ((((size_t)b * N + chunk) * Hkv + g) * C1 + slot) * cpr + c;
  const u32x4 nan4 = {kNanWord, kNanWord, kNanWord, kNanWord};
  k_sel[gid] = bad ? nan4 : k_cache[src];
  v_sel[gid] = bad ? nan4 : v_cache[src];
}

hipError_t launch_gather_selected(const void* k_cache, const void* v_cache, const int32_t* chunk_idx,
                                  const int32_t* tok_slot, void* k_sel, void* v_sel, int B, int N, int C, int Hkv,
                                  int K, int Bt, int row_bytes, hipStream_t s) {
  const int cpr = row_bytes / 16;
  const size_t total = (size_t)B * Hkv * K * (1 + Bt) * cpr;
  const dim3 grid((unsigned)((total + 255) / 256));
  hipLaunchKernelGGL(gather_selected_kernel, grid, dim3(256), 0, s, (const u32x4*)k_cache, (const u32x4*)v_cache,
                     chunk_idx, tok_slot, (u32x4*)k_sel, (u32x4*)v_sel, total, N, C + 1, Hkv, K, Bt, cpr);
  return hipGetLastError();
}

// Full-mask cache construction: the joint rows [kept rows ; L_q query rows] of
// every sequence in the decode layout [B][Lj][H][d], Q and K moved to the
// joint positions by the rotate-half rotary rotation, V copied.  Kept chunk k
// (ascending) moves by k*(C+1), the query rows by (K-1)*(C+1); element i < d/2
// pairs with i + d/2 at frequency base^(-2i/d).  The rotation runs in double
// and is rounded once to the element type.  K and V also go, when asked, to
// the compact prefix layout [B][Hkv][Lj][d] that the decoding steps read.
// One workgroup per joint row: its d/2 cosines and sines (one shift) are
// computed once into LDS, then the threads stream (tensor and head, pair of
// 16-byte chunks c and c + d/2 elements) tasks through them.
template <bool BF16>
__global__ __launch_bounds__(256) void gather_joint_kernel(JointArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;   // elements per 16-byte chunk
  __shared__ double cs_tab[64], sn_tab[64];
  const size_t jrow = blockIdx.x;     // b * Lj + j
  const int j = (int)(jrow % a.Lj), b = (int)(jrow / a.Lj);
  const int C1 = a.C + 1, n_sel = a.K * (1 + a.Bt);
  const bool kept = j < n_sel;
  int kk = a.K - 1, slot = 0;
  size_t n = 0, qm_row = 0;
  bool bad = false;
  if (kept) {
    kk = j / (1 + a.Bt);
    const int sl = j - kk * (1 + a.Bt);
    slot = sl == 0 ? 0 : a.tok_slot[((size_t)b * a.K + kk) * a.Bt + sl - 1];
    int chunk = a.chunk_idx[(size_t)b * a.K + kk];
    bad = kCheckIndices && !kept_row_ok(chunk, slot, sl == 0, a.N, a.C);
    if (bad) chunk = slot = 0;
    n = (size_t)b * a.N + chunk;
  } else {
    qm_row = (a.qm_per_chunk ? (size_t)b * a.N : (size_t)b) * (size_t)(a.Lq + a.Lm) + (j - n_sel);
  }
  const bool rot = a.rope_base > 0.0;
  if (rot) {
    const double delta = (double)kk * C1;
    for (int i = threadIdx.x; i < a.D / 2; i += 256) {
      double sn, cs;
      sincos(delta * pow(a.rope_base, -2.0 * i / a.D), &sn, &cs);
      cs_tab[i] = cs;
      sn_tab[i] = sn;
    }
    __syncthreads();
  }
  const int CP = a.D / EPC / 2;       // chunk pairs per row
  const int tasks = (a.Hq + 2 * a.Hkv) * CP;
  for (int task = threadIdx.x; task < tasks; task += 256) {
    const int cp = task % CP, th = task / CP;
    const int tensor = th < a.Hq ? 0 : (th < a.Hq + a.Hkv ? 1 : 2);   // Q, K, V
    const int head = tensor == 0 ? th : (tensor == 1 ? th - a.Hq : th - a.Hq - a.Hkv);
    const int H = tensor == 0 ? a.Hq : a.Hkv;
    size_t src_el;
    const void* src;
    if (kept) {
      if (tensor == 0) {
        src = a.q_pre;
        src_el = ((n * C1 + slot) * a.Hq + head) * a.D;
      } else {
        src = tensor == 1 ? a.k_cache : a.v_cache;
        src_el = ((n * a.Hkv + head) * C1 + slot) * a.D;
      }
    } else {
      src = tensor == 0 ? a.q_qm : (tensor == 1 ? a.k_qm : a.v_qm);
      src_el = (qm_row * H + head) * a.D;
    }
    void* dst = tensor == 0 ? a.q_joint : (tensor == 1 ? a.k_joint : a.v_joint);
    const size_t dst_el = (jrow * H + head) * a.D;
    const u32x4* s4 = reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(src) + src_el * a.elem_bytes);
    u32x4* d4 = reinterpret_cast<u32x4*>(reinterpret_cast<char*>(dst) + dst_el * a.elem_bytes);
    u32x4 lo = s4[cp], hi = s4[cp + CP];
    if (tensor < 2 && rot) {
      float x[2][EPC];
      Vec16<BF16>::load(s4 + cp, 0, x[0]);
      Vec16<BF16>::load(s4 + cp + CP, 0, x[1]);
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const int i = cp * EPC + e;   // pair index, 0 .. d/2 - 1
        const double cs = cs_tab[i], sn = sn_tab[i];
        const double p0 = x[0][e], p1 = x[1][e];
        x[0][e] = (float)(p0 * cs - p1 * sn);
        x[1][e] = (float)(p1 * cs + p0 * sn);
      }
      if constexpr (BF16) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          lo[q] = pack_bf16x2(x[0][2 * q], x[0][2 * q + 1]);
          hi[q] = pack_bf16x2(x[1][2 * q], x[1][2 * q + 1]);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          lo[q] = __float_as_uint(x[0][q]);
          hi[q] = __float_as_uint(x[1][q]);
        }
      }
    }
    if (bad) lo = hi = u32x4{kNanWord, kNanWord, kNanWord, kNanWord};
    d4[cp] = lo;
    d4[cp + CP] = hi;
    void* pref = tensor == 1 ? a.k_pref : (tensor == 2 ? a.v_pref : nullptr);
    if (pref) {
      const size_t p_el = (((size_t)b * a.Hkv + head) * a.Lj + j) * a.D;
      u32x4* p4 = reinterpret_cast<u32x4*>(reinterpret_cast<char*>(pref) + p_el * a.elem_bytes);
      p4[cp] = lo;
      p4[cp + CP] = hi;
    }
  }
}

hipError_t launch_gather_joint(const JointArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((size_t)a.B * a.Lj));
  if (a.elem_bytes == 2) hipLaunchKernelGGL(gather_joint_kernel<true>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(gather_joint_kernel<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_key_mean(const void* k_cache, float* key_mean, int B, int N, int C, int Hkv, int head_dim,
                           bool bf16, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(key_mean_kernel<true>, dim3(B * N * Hkv), dim3(256), 0, s, k_cache, key_mean, C, head_dim);
  else
    hipLaunchKernelGGL(key_mean_kernel<false>, dim3(B * N * Hkv), dim3(256), 0, s, k_cache, key_mean, C, head_dim);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Split-S merge: O = sum_s 2^(lse_s - M) O_s / sum_s 2^(lse_s - M).
template <bool BF16>
__global__ __launch_bounds__(256) void merge_kernel(const float* o_part, const float* lse_part, void* o_dec,
                                                     float* lse_dec, int S, int B, int Hq, int Ld, int D) {
  const int TPR = D / 4;
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t rows = (size_t)B * Hq * Ld;
  const size_t row = gid / TPR;
  if (row >= rows) return;
  const int c = gid % TPR;
  // Shards in groups of 8 whose loads are all issued before the first use
  // (the shard count is a run-time value); summed in ascending shard order.
  constexpr int U = 8;
  float M = -INFINITY;
  for (int s0 = 0; s0 < S; s0 += U) {
    float l[U];
#pragma unroll
    for (int u = 0; u < U; ++u) l[u] = s0 + u < S ? lse_part[(s0 + u) * rows + row] : -INFINITY;
#pragma unroll
    for (int u = 0; u < U; ++u) M = fmaxf(M, l[u]);
  }
  float W = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < S; s0 += U) {
    float l[U];
    f32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool in = s0 + u < S;
      l[u] = in ? lse_part[(s0 + u) * rows + row] : 0.f;
      v[u] = in ? *reinterpret_cast<const f32x4*>(o_part + ((s0 + u) * rows + row) * D + 4 * c) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < S) {
        const float w = fast_exp2(l[u] - M);
        W += w;
        acc += w * v[u];
      }
    }
  }
  const float inv = 1.0f / W;
  // row = (b*Hq + h)*Ld + r  ->  o_dec[b][r][h][:]
  const int r = row % Ld;
  const size_t bh = row / Ld;
  const int h = bh % Hq;
  const size_t b = bh / Hq;
  const size_t out = ((b * Ld + r) * Hq + h) * D + 4 * c;
  if constexpr (BF16) {
    u32x2 v = {pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
    *reinterpret_cast<u32x2*>(reinterpret_cast<uint16_t*>(o_dec) + out) = v;
  } else {
    *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(o_dec) + out) = acc * inv;
  }
  if (lse_dec && c == 0) lse_dec[row] = (M + __log2f(W)) * kLn2;
}

hipError_t launch_merge(const float* o_part, const float* lse_part, void* o_dec, float* lse_dec, int S, int B,
                        int Hq, int Ld, int head_dim, bool bf16, hipStream_t s) {
  const size_t threads = (size_t)B * Hq * Ld * (head_dim / 4);
  const dim3 grid((unsigned)((threads + 255) / 256));
  if (bf16)
    hipLaunchKernelGGL(merge_kernel<true>, grid, dim3(256), 0, s, o_part, lse_part, o_dec, lse_dec, S, B, Hq, Ld, head_dim);
  else
    hipLaunchKernelGGL(merge_kernel<false>, grid, dim3(256), 0, s, o_part, lse_part, o_dec, lse_dec, S, B, Hq, Ld, head_dim);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Chunk cache copy [B][N][1+C][H][d] -> [B][N][H][1+C][d], 16 bytes per thread.
__global__ __launch_bounds__(256) void cache_copy_kernel(const u32x4* k_pre, const u32x4* v_pre, u32x4* k_cache,
                                                          u32x4* v_cache, size_t total, int C1, int Hkv, int cpr) {
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= total) return;
  // source order: ((bn*C1 + s)*Hkv + g)*cpr + c
  const int c = gid % cpr;
  size_t r = gid / cpr;
  const int g = r % Hkv;
  r /= Hkv;
  const int s = r % C1;
  const size_t bn = r / C1;
  const size_t dst = ((bn * Hkv + g) * C1 + s) * cpr + c;
  k_cache[dst] = k_pre[gid];
  v_cache[dst] = v_pre[gid];
}

hipError_t launch_cache_copy(const void* k_pre, const void* v_pre, void* k_cache, void* v_cache, int B, int N, int C,
                             int Hkv, int head_dim, int elem_bytes, hipStream_t s) {
  const int cpr = head_dim * elem_bytes / 16;
  const size_t total = (size_t)B * N * (C + 1) * Hkv * cpr;
  const dim3 grid((unsigned)((total + 255) / 256));
  hipLaunchKernelGGL(cache_copy_kernel, grid, dim3(256), 0, s, (const u32x4*)k_pre, (const u32x4*)v_pre,
                     (u32x4*)k_cache, (u32x4*)v_cache, total, C + 1, Hkv, cpr);
  return hipGetLastError();
}

}  // namespace pd
