// bf16 attention kernels for gfx950: chunk prefill (stage a) and sparse decode
// attention (stage c).  Both run one tile engine:
//
//   * a workgroup = 4 waves = 128 query rows (32 per wave), d = 64 or 128;
//   * K/V tiles of 64 rows are staged through LDS (K row-major, V transposed);
//   * S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_32x32x16_bf16 with
//     fp32 accumulation; Q stays in registers for the whole sweep;
//   * online softmax in the log2 domain, lazy rescaling of the running output
//     (only when a row maximum grows by more than 2^8), P rounded to bf16.
//
// Computing S transposed makes the MFMA output layout (each lane: one query,
// 16 keys) directly usable as the B operand of the P*V product: the keys a
// lane holds become its contraction slice, and the V^T operand is read in the
// same key order by storing V^T in LDS with key bits 2 and 3 swapped.
#include "pd_common.h"
#include "pd_kernels.h"

namespace pd {

template <int D>
struct Tile {
  static constexpr int BM = 128;             // query rows per workgroup
  static constexpr int BN = 64;              // key rows per KV tile
  static constexpr int NT = 256;             // threads per workgroup
  static constexpr int CH = D / 8;           // 16-byte chunks per row
  static constexpr int RPT = BN * CH / NT;   // rows each thread stages per tile
  static constexpr int KS = D / 16;          // MFMA k-steps along d
  static constexpr int DB = D / 32;          // 32-row blocks of O^T
  static constexpr int KPAD = D + 8;         // K row stride in LDS (elements)
  static constexpr int VPAD = BN + 8;        // V^T row stride in LDS (elements)
  static_assert(RPT == 2 || RPT == 4, "unsupported head dim");
};

// Column of key k (0..63) inside a V^T row: bits 2 and 3 swapped, so that the
// 8 keys one lane contracts over in a k-step are 16 contiguous bytes.
__device__ __forceinline__ int vt_col(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Engine state of one wave: 32 query rows.
template <int D>
struct WaveState {
  bf16x8 qf[Tile<D>::KS];
  f32x16 o[Tile<D>::DB];
  float m;      // running row max (log2 domain), shared by lanes l and l^32
  float l;      // this lane's partial row sum
  float qmass;  // this lane's partial mass on the query columns (prefill only)
};

// Stage one K/V tile held in registers into LDS.
template <int D>
__device__ __forceinline__ void stage_tile(uint16_t* Ks, uint16_t* Vt, int rg, int c,
                                           const u32x4 (&kr)[Tile<D>::RPT],
                                           const u32x4 (&vr)[Tile<D>::RPT]) {
  using T = Tile<D>;
#pragma unroll
  for (int i = 0; i < T::RPT; ++i) st16(Ks + (rg * T::RPT + i) * T::KPAD + 8 * c, kr[i]);
  const int col = vt_col(rg * T::RPT);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int w = e >> 1, sh = (e & 1) * 16;
    uint32_t h0 = (vr[0][w] >> sh) & 0xffffu;
    uint32_t h1 = (vr[1][w] >> sh) & 0xffffu;
    uint16_t* dst = Vt + (8 * c + e) * T::VPAD + col;
    if constexpr (T::RPT == 4) {
      uint32_t h2 = (vr[2][w] >> sh) & 0xffffu;
      uint32_t h3 = (vr[3][w] >> sh) & 0xffffu;
      u32x2 v = {h0 | (h1 << 16), h2 | (h3 << 16)};
      *reinterpret_cast<u32x2*>(dst) = v;
    } else {
      *reinterpret_cast<uint32_t*>(dst) = h0 | (h1 << 16);
    }
  }
}

// One KV tile for one wave: S^T = K Q^T, online softmax, O^T += V^T P^T.
// kv_valid: number of valid keys in this tile (64 except in a ragged last tile).
// qlo/qhi: key range (tile-relative) counted into qmass; empty when qlo >= qhi.
template <int D>
__device__ __forceinline__ void tile_step(WaveState<D>& st, const uint16_t* Ks, const uint16_t* Vt,
                                          int l32, int grp, float scale_log2, int kv_valid,
                                          int qlo, int qhi) {
  using T = Tile<D>;
  f32x16 s[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) s[kb] = f32x16{0};
#pragma unroll
  for (int ks = 0; ks < T::KS; ++ks) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 a = __builtin_bit_cast(bf16x8, ld16(Ks + (32 * kb + l32) * T::KPAD + 16 * ks + 8 * grp));
      s[kb] = mfma32x32x16(a, st.qf[ks], s[kb]);
    }
  }
  // Key of s[kb][r]: 32*kb + 8*(r/4) + 4*grp + r%4.
  float mx = -INFINITY;
  if (kv_valid >= 64) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[kb][r] *= scale_log2;
        mx = fmaxf(mx, s[kb][r]);
      }
  } else {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + 8 * (r >> 2) + 4 * grp + (r & 3);
        s[kb][r] = key < kv_valid ? s[kb][r] * scale_log2 : -INFINITY;
        mx = fmaxf(mx, s[kb][r]);
      }
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const bool upd = mx > st.m + 8.0f;
  if (__ballot(upd)) {
    const float mnew = upd ? mx : st.m;
    const float alpha = fast_exp2(st.m - mnew);
    st.m = mnew;
    st.l *= alpha;
    st.qmass *= alpha;
#pragma unroll
    for (int db = 0; db < T::DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[db][r] *= alpha;
  }
  bf16x8 pf[4];
  float lsum = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float pv = fast_exp2(s[kb][r] - st.m);
      s[kb][r] = pv;
      lsum += pv;
      pf[2 * kb + (r >> 3)][r & 7] = (__bf16)pv;
    }
  st.l += lsum;
  if (qlo < qhi) {
    float qs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + 8 * (r >> 2) + 4 * grp + (r & 3);
        qs += (key >= qlo && key < qhi) ? s[kb][r] : 0.f;
      }
    st.qmass += qs;
  }
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
    for (int db = 0; db < T::DB; ++db) {
      bf16x8 a = __builtin_bit_cast(bf16x8, ld16(Vt + (32 * db + l32) * T::VPAD + 16 * kk + 8 * grp));
      st.o[db] = mfma32x32x16(a, pf[kk], st.o[db]);
    }
  }
}

template <int D>
__device__ __forceinline__ void wave_init(WaveState<D>& st) {
#pragma unroll
  for (int db = 0; db < Tile<D>::DB; ++db) st.o[db] = f32x16{0};
  st.m = -INFINITY;
  st.l = 0.f;
  st.qmass = 0.f;
}

// Normalised O^T of this lane (query l32) for d = 32*db + 8*i + 4*grp + j is
// st.o[db][4*i+j] * inv; store one row of D bf16 values.
template <int D>
__device__ __forceinline__ void store_row_bf16(uint16_t* dst, const WaveState<D>& st, float inv, int grp) {
#pragma unroll
  for (int db = 0; db < Tile<D>::DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u32x2 v = {pack_bf16x2(st.o[db][4 * i] * inv, st.o[db][4 * i + 1] * inv),
                 pack_bf16x2(st.o[db][4 * i + 2] * inv, st.o[db][4 * i + 3] * inv)};
      *reinterpret_cast<u32x2*>(dst + 32 * db + 8 * i + 4 * grp) = v;
    }
}

template <int D>
__device__ __forceinline__ void store_row_f32(float* dst, const WaveState<D>& st, float inv, int grp) {
#pragma unroll
  for (int db = 0; db < Tile<D>::DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f32x4 v = {st.o[db][4 * i] * inv, st.o[db][4 * i + 1] * inv, st.o[db][4 * i + 2] * inv,
                 st.o[db][4 * i + 3] * inv};
      *reinterpret_cast<f32x4*>(dst + 32 * db + 8 * i + 4 * grp) = v;
    }
}

// ---------------------------------------------------------------------------
// Stage (a): chunk prefill.  Workgroup = (b, n, h, 128-row query tile).
// Also writes the chunk KV cache (each KV tile by exactly one workgroup of the
// (b, n, kv-head) group), the per-head query-column mass of the content rows
// and the log2-domain LSE of the query rows.
template <int D>
__global__ __launch_bounds__(256) void prefill_bf16_kernel(PrefillArgs p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[T::BN * T::KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * T::VPAD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, grp = lane >> 5;
  int lid = xcd_remap(blockIdx.x, p.total);
  const int qt = lid % p.n_qt;
  lid /= p.n_qt;
  const int h = lid % p.Hq;
  lid /= p.Hq;
  const int n = lid % p.N;
  const int b = lid / p.N;
  const int g = h / p.G;
  const int C1 = p.C + 1;
  const size_t chunk = (size_t)b * p.N + n;
  const size_t qm_base = (p.qm_per_chunk ? chunk : (size_t)b) * (size_t)(p.Lq + p.Lm);

  // Q fragment of this lane's query row.
  WaveState<D> st;
  const int qrow = qt * T::BM + wave * 32 + l32;
  const bool wave_active = qt * T::BM + wave * 32 < p.Sc;
  {
    const uint16_t* src = nullptr;
    if (qrow < C1) src = p.q_pre + ((chunk * C1 + qrow) * p.Hq + h) * D;
    else if (qrow < p.Sc) src = p.q_qm + ((qm_base + (qrow - C1)) * p.Hq + h) * D;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks)
      st.qf[ks] = src ? __builtin_bit_cast(bf16x8, ld16(src + 16 * ks + 8 * grp)) : bf16x8{0};
  }
  wave_init(st);

  const int c = tid % T::CH, rg = tid / T::CH;
  u32x4 kr[T::RPT], vr[T::RPT];
  auto load = [&](int t) {
#pragma unroll
    for (int i = 0; i < T::RPT; ++i) {
      const int row = t * T::BN + rg * T::RPT + i;
      if (row < C1) {
        const size_t off = ((chunk * C1 + row) * p.Hkv + g) * D + 8 * c;
        kr[i] = ld16(p.k_pre + off);
        vr[i] = ld16(p.v_pre + off);
      } else if (row < p.Sc) {
        const size_t off = ((qm_base + (row - C1)) * p.Hkv + g) * D + 8 * c;
        kr[i] = ld16(p.k_qm + off);
        vr[i] = ld16(p.v_qm + off);
      } else {
        kr[i] = u32x4{0, 0, 0, 0};
        vr[i] = u32x4{0, 0, 0, 0};
      }
    }
  };
  auto cache_write = [&](int t) {
    const bool writer = (t % p.n_qt == qt) && ((t / p.n_qt) % p.G == h % p.G);
    if (!writer) return;
#pragma unroll
    for (int i = 0; i < T::RPT; ++i) {
      const int row = t * T::BN + rg * T::RPT + i;
      if (row < C1) {
        const size_t off = (((chunk * p.Hkv + g) * C1) + row) * D + 8 * c;
        st16(p.k_cache + off, kr[i]);
        st16(p.v_cache + off, vr[i]);
      }
    }
  };

  const int qc_lo = C1, qc_hi = C1 + p.Lq;   // query columns counted by Eq. 5
  load(0);
  cache_write(0);
  stage_tile<D>(Ks, Vt, rg, c, kr, vr);
  __syncthreads();
  for (int t = 0; t < p.n_kvt; ++t) {
    if (t + 1 < p.n_kvt) load(t + 1);
    if (wave_active) {
      const int t0 = t * T::BN;
      const int kv_valid = min(T::BN, p.Sc - t0);
      const int lo = max(qc_lo - t0, 0), hi = min(qc_hi - t0, T::BN);
      tile_step<D>(st, Ks, Vt, l32, grp, p.scale_log2, kv_valid, lo, hi);
    }
    __syncthreads();
    if (t + 1 < p.n_kvt) {
      cache_write(t + 1);
      stage_tile<D>(Ks, Vt, rg, c, kr, vr);
    }
    __syncthreads();
  }
  if (!wave_active) return;

  const float ltot = st.l + __shfl_xor(st.l, 32);
  const float qtot = st.qmass + __shfl_xor(st.qmass, 32);
  const float inv = 1.0f / ltot;
  if (qrow < p.Sc) {
    uint16_t* dst = p.o + ((chunk * p.Sc + qrow) * p.Hq + h) * D;
    store_row_bf16<D>(dst, st, inv, grp);
    if (grp == 0) {
      const size_t hb = chunk * p.Hq + h;
      if (qrow >= 1 && qrow < C1) p.part_i[hb * p.C + (qrow - 1)] = qtot * inv;
      if (qrow >= qc_lo && qrow < qc_hi) p.lse_q[hb * p.Lq + (qrow - qc_lo)] = st.m + __log2f(ltot);
    }
  }
}

// ---------------------------------------------------------------------------
// Stage (c): sparse decode attention.  Workgroup = (b, kv head g, 128-row tile
// of the G*L_d query rows of that group, KV shard).  Query row rho of the group
// is head g*G + rho / L_d, decode row rho % L_d.  KV row j of the shard walks:
// [kept chunks: BOS + kept slots] ; [static rows] ; [own rows].
template <int D>
__global__ __launch_bounds__(256) void decode_bf16_kernel(DecodeArgs p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[T::BN * T::KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * T::VPAD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, grp = lane >> 5;
  int lid = xcd_remap(blockIdx.x, p.total);
  const int sp = lid % p.S;
  lid /= p.S;
  const int qt = lid % p.n_qt;
  lid /= p.n_qt;
  const int g = lid % p.Hkv;
  const int b = lid / p.Hkv;
  const int GL = p.G * p.Ld;
  const int C1 = p.C + 1;
  const int n_sel = p.K * (1 + p.Bt);
  const int L_kv = n_sel + p.n_static + p.Ld;

  WaveState<D> st;
  const int rho = qt * T::BM + wave * 32 + l32;
  const bool wave_active = qt * T::BM + wave * 32 < GL;
  const int hq = g * p.G + (rho < GL ? rho / p.Ld : 0);
  const int rr = rho < GL ? rho % p.Ld : 0;
  {
    const uint16_t* src = rho < GL ? p.q_dec + (((size_t)b * p.Ld + rr) * p.Hq + hq) * D : nullptr;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks)
      st.qf[ks] = src ? __builtin_bit_cast(bf16x8, ld16(src + 16 * ks + 8 * grp)) : bf16x8{0};
  }
  wave_init(st);

  // This shard's tiles.
  const int n_kvt = (L_kv + T::BN - 1) / T::BN;
  const int t_begin = (int)(((long long)n_kvt * sp) / p.S);
  const int t_end = (int)(((long long)n_kvt * (sp + 1)) / p.S);

  const int c = tid % T::CH, rg = tid / T::CH;
  const size_t cache_bg = ((size_t)b * p.N * p.Hkv + g) * C1;   // + (n*Hkv)*C1 + slot
  const int32_t* cidx = p.chunk_idx + (size_t)b * p.K;
  const int32_t* tslot = p.tok_slot + (size_t)b * p.K * p.Bt;
  u32x4 kr[T::RPT], vr[T::RPT];
  auto load = [&](int t) {
#pragma unroll
    for (int i = 0; i < T::RPT; ++i) {
      const int j = t * T::BN + rg * T::RPT + i;
      const uint16_t *ks = nullptr, *vs = nullptr;
      size_t off = 0;
      if (j < n_sel) {
        const int kk = j / (1 + p.Bt), s = j - kk * (1 + p.Bt);
        const int nn = cidx[kk];
        const int slot = s == 0 ? 0 : tslot[kk * p.Bt + s - 1];
        off = (cache_bg + (size_t)nn * p.Hkv * C1 + slot) * D;
        ks = p.k_cache;
        vs = p.v_cache;
      } else if (j < n_sel + p.n_static) {
        off = (((size_t)b * p.Ls + (j - n_sel)) * p.Hkv + g) * D;
        ks = p.k_static;
        vs = p.v_static;
      } else if (j < L_kv) {
        off = (((size_t)b * p.Ld + (j - n_sel - p.n_static)) * p.Hkv + g) * D;
        ks = p.k_dec;
        vs = p.v_dec;
      }
      if (ks) {
        kr[i] = ld16(ks + off + 8 * c);
        vr[i] = ld16(vs + off + 8 * c);
      } else {
        kr[i] = u32x4{0, 0, 0, 0};
        vr[i] = u32x4{0, 0, 0, 0};
      }
    }
  };

  load(t_begin);
  stage_tile<D>(Ks, Vt, rg, c, kr, vr);
  __syncthreads();
  for (int t = t_begin; t < t_end; ++t) {
    if (t + 1 < t_end) load(t + 1);
    if (wave_active) {
      const int kv_valid = min(T::BN, L_kv - t * T::BN);
      tile_step<D>(st, Ks, Vt, l32, grp, p.scale_log2, kv_valid, 0, 0);
    }
    __syncthreads();
    if (t + 1 < t_end) stage_tile<D>(Ks, Vt, rg, c, kr, vr);
    __syncthreads();
  }
  if (!wave_active || rho >= GL) return;

  const float ltot = st.l + __shfl_xor(st.l, 32);
  const float inv = 1.0f / ltot;
  const float lse2 = st.m + __log2f(ltot);
  if (p.S == 1) {
    uint16_t* dst = reinterpret_cast<uint16_t*>(p.o_dec) + (((size_t)b * p.Ld + rr) * p.Hq + hq) * D;
    store_row_bf16<D>(dst, st, inv, grp);
    if (p.lse_dec && grp == 0) p.lse_dec[((size_t)b * p.Hq + hq) * p.Ld + rr] = lse2 * kLn2;
  } else {
    const size_t row = (((size_t)sp * p.B + b) * p.Hq + hq) * p.Ld + rr;
    store_row_f32<D>(p.o_part + row * D, st, inv, grp);
    if (grp == 0) p.lse_part[row] = lse2;
  }
}

// ---------------------------------------------------------------------------
// Eq. 5, second sum: for each content token j, the softmax mass the L_q query
// rows put on it, summed over heads, plus the first sum (per-head query-column
// mass of row j, written by the prefill kernel).  Workgroup = (b, n, 64 content
// columns); wave w handles heads w, w+4, ...  S = Q_q K_c^T on MFMA, then
// exp2(S*scale - lse2(row)) with the query rows' final LSE from the prefill.
template <int D>
__global__ __launch_bounds__(256) void escore_bf16_kernel(EscoreArgs p) {
  constexpr int KS = D / 16;
  __shared__ float red[4][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, grp = lane >> 5;
  int lid = blockIdx.x;
  const int cb = lid % p.n_cb;
  lid /= p.n_cb;
  const int n = lid % p.N;
  const int b = lid / p.N;
  const int C1 = p.C + 1;
  const size_t chunk = (size_t)b * p.N + n;
  const size_t qm_base = (p.qm_per_chunk ? chunk : (size_t)b) * (size_t)(p.Lq + p.Lm);
  const int n_qb = (p.Lq + 31) / 32;

  float colsum[2] = {0.f, 0.f};
  for (int h = wave; h < p.Hq; h += 4) {
    const int g = h / p.G;
    bf16x8 kf[2][KS];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int j = cb * 64 + 32 * kb + l32;
      const uint16_t* src = j < p.C ? p.k_cache + ((chunk * p.Hkv + g) * C1 + 1 + j) * D : nullptr;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kf[kb][ks] = src ? __builtin_bit_cast(bf16x8, ld16(src + 16 * ks + 8 * grp)) : bf16x8{0};
    }
    const float* lse = p.lse_q + (chunk * p.Hq + h) * p.Lq;
    for (int qb = 0; qb < n_qb; ++qb) {
      const int qrow = qb * 32 + l32;
      const uint16_t* qsrc = qrow < p.Lq ? p.q_qm + ((qm_base + qrow) * p.Hq + h) * D : nullptr;
      bf16x8 qa[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qa[ks] = qsrc ? __builtin_bit_cast(bf16x8, ld16(qsrc + 16 * ks + 8 * grp)) : bf16x8{0};
      // Row (query) of element r: qb*32 + 8*(r/4) + 4*grp + r%4.
      float lrow[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int q = qb * 32 + 8 * (r >> 2) + 4 * grp + (r & 3);
        lrow[r] = q < p.Lq ? lse[q] : INFINITY;
      }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = f32x16{0};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) s = mfma32x32x16(qa[ks], kf[kb][ks], s);
        float acc = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc += fast_exp2(s[r] * p.scale_log2 - lrow[r]);
        colsum[kb] += acc;
      }
    }
  }
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const float v = colsum[kb] + __shfl_xor(colsum[kb], 32);
    if (grp == 0) red[wave][32 * kb + l32] = v;
  }
  __syncthreads();
  if (tid < 64) {
    const int j = cb * 64 + tid;
    if (j < p.C) {
      float e = 0.f;
      for (int h = 0; h < p.Hq; ++h) e += p.part_i[(chunk * p.Hq + h) * p.C + j];
      e += ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
      p.tok_score[chunk * p.C + j] = e;
    }
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers.
template <int D>
static hipError_t launch_prefill_d(const PrefillArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(prefill_bf16_kernel<D>, dim3(a.total), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_prefill_bf16(const PrefillArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? launch_prefill_d<128>(a, s) : launch_prefill_d<64>(a, s);
}

template <int D>
static hipError_t launch_decode_d(const DecodeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(decode_bf16_kernel<D>, dim3(a.total), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_decode_bf16(const DecodeArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? launch_decode_d<128>(a, s) : launch_decode_d<64>(a, s);
}

template <int D>
static hipError_t launch_escore_d(const EscoreArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(escore_bf16_kernel<D>, dim3(a.total), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_escore_bf16(const EscoreArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? launch_escore_d<128>(a, s) : launch_escore_d<64>(a, s);
}

}  // namespace pd
