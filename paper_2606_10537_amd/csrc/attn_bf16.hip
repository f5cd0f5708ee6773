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
  float l;      // this lane's partial sum of the bf16-rounded weights that multiply V
  float lx;     // this lane's partial sum of the unrounded weights (prefill only)
  float qmass;  // this lane's partial mass on the query columns (prefill only)
};

// Thread -> (row group, 16-byte chunk) mappings used to stage a 64-row tile.
// K: thread t takes chunk t % CH of rows RPT*(t / CH) .. +RPT-1 (row-major
// stores, every bank hit equally often).  V: each wave takes all row groups
// and CH/4 chunks, so that the 8 transposed stores of a thread (V^T rows 8c+e)
// from one wave land on V^T rows whose 36-dword-strided bases alternate bank
// halves: every bank is hit exactly twice per store instruction.
template <int D>
struct StageMap {
  int rgk, ck, rgv, cv;
  __device__ StageMap(int tid) {
    using T = Tile<D>;
    const int lane = tid & 63, wave = tid >> 6, cpw = T::CH / 4;
    ck = tid % T::CH;
    rgk = tid / T::CH;
    rgv = lane / cpw;
    cv = wave * cpw + lane % cpw;
  }
};

// Stage one K/V tile held in registers into LDS.
template <int D>
__device__ __forceinline__ void stage_tile(uint16_t* Ks, uint16_t* Vt, const StageMap<D>& mp,
                                           const u32x4 (&kr)[Tile<D>::RPT],
                                           const u32x4 (&vr)[Tile<D>::RPT]) {
  using T = Tile<D>;
#pragma unroll
  for (int i = 0; i < T::RPT; ++i) st16(Ks + (mp.rgk * T::RPT + i) * T::KPAD + 8 * mp.ck, kr[i]);
  const int col = vt_col(mp.rgv * T::RPT);
  // Element e of each of the RPT rows, packed two halves per v_perm_b32:
  // selector 0x05040100 takes the low halves of (lo, hi), 0x07060302 the high.
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int w = e >> 1;
    const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
    uint16_t* dst = Vt + (8 * mp.cv + e) * T::VPAD + col;
    const uint32_t a = __builtin_amdgcn_perm(vr[1][w], vr[0][w], sel);
    if constexpr (T::RPT == 4) {
      const uint32_t b = __builtin_amdgcn_perm(vr[3][w], vr[2][w], sel);
      *reinterpret_cast<u32x2*>(dst) = u32x2{a, b};
    } else {
      *reinterpret_cast<uint32_t*>(dst) = a;
    }
  }
}

// One KV tile for one wave: S^T = K Q^T, online softmax, O^T += V^T P^T.
// kv_valid: number of valid keys in this tile (64 except in a ragged last tile).
// qlo/qhi: key range (tile-relative) counted into qmass; empty when qlo >= qhi.
// EXACT: also keep the unrounded row sum and the query-column mass (prefill).
// O is normalised by the sum of the same bf16-rounded weights that multiply V,
// so rounding P perturbs a convex combination instead of scaling O.
template <int D, bool EXACT>
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
  // Key of s[kb][r]: 32*kb + 8*(r/4) + 4*grp + r%4.  The max is taken on raw
  // scores (the scale is positive) and the scale is folded into one FMA:
  // p = exp2(s * scale_log2 - m).
  if (kv_valid < 64) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + 8 * (r >> 2) + 4 * grp + (r & 3);
        s[kb][r] = key < kv_valid ? s[kb][r] : -INFINITY;
      }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; r += 2) mx = fmaxf(mx, fmaxf(s[kb][r], s[kb][r + 1]));
  mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;
  const bool upd = mx > st.m + 8.0f;
  if (__ballot(upd)) {
    const float mnew = upd ? mx : st.m;
    const float alpha = fast_exp2(st.m - mnew);
    st.m = mnew;
    st.l *= alpha;
    if constexpr (EXACT) {
      st.lx *= alpha;
      st.qmass *= alpha;
    }
#pragma unroll
    for (int db = 0; db < T::DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) st.o[db][r] *= alpha;
  }
  const float nm = -st.m;
  uint32_t pk[16];
  float lsum = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
      const float p0 = fast_exp2(fmaf(s[kb][r], scale_log2, nm));
      const float p1 = fast_exp2(fmaf(s[kb][r + 1], scale_log2, nm));
      s[kb][r] = p0;
      s[kb][r + 1] = p1;
      if constexpr (EXACT) lsum += p0 + p1;
      pk[8 * kb + r / 2] = __builtin_bit_cast(uint32_t, bf16x2{(__bf16)p0, (__bf16)p1});
    }
  if constexpr (EXACT) st.lx += lsum;
  // Sum of the rounded weights: one v_dot2c_f32_bf16 with (1, 1) per packed pair.
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float lr = st.l;
#pragma unroll
  for (int i = 0; i < 16; ++i) lr = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[i]), ones, lr, false);
  st.l = lr;
  bf16x8 pf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
    pf[kk] = __builtin_bit_cast(bf16x8, u32x4{pk[4 * kk], pk[4 * kk + 1], pk[4 * kk + 2], pk[4 * kk + 3]});
  if (EXACT && qlo < qhi) {
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
  st.lx = 0.f;
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

// Double-buffered sweep over KV tiles [t_begin, t_end): tile t is computed from
// LDS buffer (t - t_begin) & 1 while tile t+1 is staged into the other buffer
// and tile t+2 is already loading into registers; one barrier per tile.
// load(t, kr, vr) fills the registers, hook(t, kr, vr) sees them before staging
// (the prefill writes its cache share there), step(t, Ks, Vt) computes.
template <int D, class Load, class Hook, class Step>
__device__ __forceinline__ void kv_sweep(uint16_t* Ks0, uint16_t* Vt0, int t_begin, int t_end, const StageMap<D>& mp,
                                         Load&& load, Hook&& hook, Step&& step) {
  using T = Tile<D>;
  constexpr int KSZ = T::BN * T::KPAD, VSZ = D * T::VPAD;
  u32x4 kr[T::RPT], vr[T::RPT];
  load(t_begin, kr, vr);
  hook(t_begin, kr, vr);
  stage_tile<D>(Ks0, Vt0, mp, kr, vr);
  if (t_begin + 1 < t_end) load(t_begin + 1, kr, vr);
  __syncthreads();
  for (int t = t_begin; t < t_end; ++t) {
    const int cur = (t - t_begin) & 1;
    step(t, Ks0 + cur * KSZ, Vt0 + cur * VSZ);
    if (t + 1 < t_end) {
      hook(t + 1, kr, vr);
      stage_tile<D>(Ks0 + (cur ^ 1) * KSZ, Vt0 + (cur ^ 1) * VSZ, mp, kr, vr);
      if (t + 2 < t_end) load(t + 2, kr, vr);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Stage (a): chunk prefill.  Workgroup = (b, n, h, 128-row query tile).
// Also writes the chunk KV cache (each KV tile by exactly one workgroup of the
// (b, n, kv-head) group), the per-head query-column mass of the content rows
// and the log2-domain LSE of the query rows.
template <int D>
__global__ __launch_bounds__(256, 2) void prefill_bf16_kernel(PrefillArgs p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2 * T::BN * T::KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2 * D * T::VPAD];

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

  const StageMap<D> mp(tid);
  // Row r of the chunk sequence lives at base + r*HD (HD = H_kv*d elements), with
  // base the chunk's rows for r <= C and the shared query/pseudo-label rows after.
  // Rows past the end are clamped to the last row: their keys are masked out of
  // the softmax and their (finite) values get probability 0.
  const int HD = p.Hkv * D;
  const uint16_t* k_lo = p.k_pre + (chunk * C1 * p.Hkv + g) * D;
  const uint16_t* v_lo = p.v_pre + (chunk * C1 * p.Hkv + g) * D;
  const uint16_t* k_hi = p.k_qm + (qm_base * p.Hkv + g) * D - (size_t)C1 * HD;
  const uint16_t* v_hi = p.v_qm + (qm_base * p.Hkv + g) * D - (size_t)C1 * HD;
  const int offk = mp.rgk * T::RPT * HD + 8 * mp.ck;   // this thread's first K row, within a tile
  const int offv = mp.rgv * T::RPT * HD + 8 * mp.cv;
  auto load = [&](int t, u32x4 (&kr)[T::RPT], u32x4 (&vr)[T::RPT]) {
    const int r0 = t * T::BN;
    if (r0 + T::BN <= C1 || (r0 >= C1 && r0 + T::BN <= p.Sc)) {
      // Whole tile inside one source: rows r0.. at base + r0*HD, no per-row selects.
      const uint16_t* kb = (r0 < C1 ? k_lo : k_hi) + (size_t)r0 * HD;
      const uint16_t* vb = (r0 < C1 ? v_lo : v_hi) + (size_t)r0 * HD;
#pragma unroll
      for (int i = 0; i < T::RPT; ++i) {
        kr[i] = ld16(kb + (unsigned)(offk + i * HD));
        vr[i] = ld16(vb + (unsigned)(offv + i * HD));
      }
    } else {
#pragma unroll
      for (int i = 0; i < T::RPT; ++i) {
        const int rk = min(r0 + mp.rgk * T::RPT + i, p.Sc - 1);
        const int rv = min(r0 + mp.rgv * T::RPT + i, p.Sc - 1);
        kr[i] = ld16((rk < C1 ? k_lo : k_hi) + (unsigned)(rk * HD + 8 * mp.ck));
        vr[i] = ld16((rv < C1 ? v_lo : v_hi) + (unsigned)(rv * HD + 8 * mp.cv));
      }
    }
  };
  // Each KV tile of the (b, n, kv head) group is written to the cache by exactly
  // one workgroup of that group: query tile t % n_qt of head g*G + (t / n_qt) % G.
  auto cache_write = [&](int t, const u32x4 (&kr)[T::RPT], const u32x4 (&vr)[T::RPT]) {
    const bool writer = (t % p.n_qt == qt) && ((t / p.n_qt) % p.G == h % p.G);
    if (!writer) return;
    const size_t base = (chunk * p.Hkv + g) * C1;
#pragma unroll
    for (int i = 0; i < T::RPT; ++i) {
      const int rk = t * T::BN + mp.rgk * T::RPT + i;
      if (rk < C1) st16(p.k_cache + (base + rk) * D + 8 * mp.ck, kr[i]);
      const int rv = t * T::BN + mp.rgv * T::RPT + i;
      if (rv < C1) st16(p.v_cache + (base + rv) * D + 8 * mp.cv, vr[i]);
    }
  };

  const int qc_lo = C1, qc_hi = C1 + p.Lq;   // query columns counted by Eq. 5
  kv_sweep<D>(Ks, Vt, 0, p.n_kvt, mp, load, cache_write, [&](int t, const uint16_t* ks, const uint16_t* vt) {
    if (!wave_active) return;
    const int t0 = t * T::BN;
    const int kv_valid = min(T::BN, p.Sc - t0);
    const int lo = max(qc_lo - t0, 0), hi = min(qc_hi - t0, T::BN);
    tile_step<D, true>(st, ks, vt, l32, grp, p.scale_log2, kv_valid, lo, hi);
  });
  if (!wave_active) return;

  const float ltot = st.l + __shfl_xor(st.l, 32);
  const float lxtot = st.lx + __shfl_xor(st.lx, 32);
  const float qtot = st.qmass + __shfl_xor(st.qmass, 32);
  const float inv = 1.0f / ltot;
  if (qrow < p.Sc) {
    const size_t orow = ((chunk * p.Sc + qrow) * p.Hq + h) * D;
    if (p.out_f32) store_row_f32<D>(reinterpret_cast<float*>(p.o) + orow, st, inv, grp);
    else store_row_bf16<D>(p.o + orow, st, inv, grp);
    if (grp == 0) {
      const size_t hb = chunk * p.Hq + h;
      if (qrow >= 1 && qrow < C1) p.part_i[hb * p.C + (qrow - 1)] = qtot / lxtot;
      if (qrow >= qc_lo && qrow < qc_hi) p.lse_q[hb * p.Lq + (qrow - qc_lo)] = st.m + __log2f(lxtot);
    }
  }
}

// ---------------------------------------------------------------------------
// Stage (c): sparse decode attention.  Workgroup = (b, kv head g, 128-row tile
// of the G*L_d query rows of that group, KV shard).  Query row rho of the group
// is head g*G + rho / L_d, decode row rho % L_d.  KV row j of the shard walks:
// [kept chunks: BOS + kept slots] ; [static rows] ; [own rows].
template <int D>
__global__ __launch_bounds__(256, 2) void decode_bf16_kernel(DecodeArgs p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2 * T::BN * T::KPAD];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2 * D * T::VPAD];
  __shared__ __attribute__((aligned(16))) int rowtab[kDecodeTableRows];   // cache row (n*Hkv*(C+1) + slot) of gathered rows

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

  const StageMap<D> mp(tid);
  const size_t cache_bg = ((size_t)b * p.N * p.Hkv + g) * C1;   // + n*Hkv*C1 + slot
  // Gathered rows of this shard: row codes into LDS once (the host keeps every
  // shard within kDecodeTableRows rows), so tile loads need no index fetch.
  const int j_lo = t_begin * T::BN;
  const int j_hi = min(t_end * T::BN, n_sel);
  {
    const int32_t* cidx = p.chunk_idx + (size_t)b * p.K;
    const int32_t* tslot = p.tok_slot + (size_t)b * p.K * p.Bt;
    for (int j = j_lo + tid; j < j_hi; j += T::NT) {
      const int kk = j / (1 + p.Bt), s = j - kk * (1 + p.Bt);
      const int slot = s == 0 ? 0 : tslot[kk * p.Bt + s - 1];
      rowtab[j - j_lo] = cidx[kk] * p.Hkv * C1 + slot;
    }
  }
  __syncthreads();
  // Row j of the shard: gathered cache rows (offset from the LDS table), then
  // static rows, then own rows, each at base + row*HD for the latter two.  Rows
  // past L_kv are clamped to the last row (masked out of the softmax).
  const int HD = p.Hkv * D;
  const uint16_t* kc = p.k_cache + cache_bg * D;
  const uint16_t* vc = p.v_cache + cache_bg * D;
  const size_t sb = ((size_t)b * p.Ls * p.Hkv + g) * D - (size_t)n_sel * HD;
  const size_t db = ((size_t)b * p.Ld * p.Hkv + g) * D - (size_t)(n_sel + p.n_static) * HD;
  const uint16_t* ks_ = p.k_static ? p.k_static + sb : p.k_dec + db;
  const uint16_t* vs_ = p.v_static ? p.v_static + sb : p.v_dec + db;
  const uint16_t* kd_ = p.k_dec + db;
  const uint16_t* vd_ = p.v_dec + db;
  const int tab_hi = max(j_hi - j_lo - 1, 0);
  auto row_ptr = [&](int j, const uint16_t* c_, const uint16_t* s_, const uint16_t* d_, int ch) {
    j = min(j, L_kv - 1);
    const unsigned tab = (unsigned)rowtab[min(max(j - j_lo, 0), tab_hi)] * D;
    const uint16_t* base = j < n_sel ? c_ : (j < n_sel + p.n_static ? s_ : d_);
    const unsigned off = j < n_sel ? tab : (unsigned)(j * HD);
    return base + off + 8 * ch;
  };
  static_assert(T::RPT == 4 || T::RPT == 2, "");
  auto load = [&](int t, u32x4 (&kr)[T::RPT], u32x4 (&vr)[T::RPT]) {
    const int r0 = t * T::BN;
    if (r0 + T::BN <= n_sel) {
      // Whole tile gathered from the cache: the RPT row codes of a thread are
      // consecutive table entries (one LDS read).
      const int* tk = rowtab + (r0 - j_lo) + mp.rgk * T::RPT;
      const int* tv = rowtab + (r0 - j_lo) + mp.rgv * T::RPT;
      int ck[T::RPT], cv[T::RPT];
      if constexpr (T::RPT == 4) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(tk), b = *reinterpret_cast<const u32x4*>(tv);
#pragma unroll
        for (int i = 0; i < 4; ++i) { ck[i] = (int)a[i]; cv[i] = (int)b[i]; }
      } else {
        const u32x2 a = *reinterpret_cast<const u32x2*>(tk), b = *reinterpret_cast<const u32x2*>(tv);
#pragma unroll
        for (int i = 0; i < 2; ++i) { ck[i] = (int)a[i]; cv[i] = (int)b[i]; }
      }
#pragma unroll
      for (int i = 0; i < T::RPT; ++i) {
        kr[i] = ld16(kc + ((unsigned)ck[i] * D + 8 * mp.ck));
        vr[i] = ld16(vc + ((unsigned)cv[i] * D + 8 * mp.cv));
      }
    } else {
#pragma unroll
      for (int i = 0; i < T::RPT; ++i) {
        kr[i] = ld16(row_ptr(r0 + mp.rgk * T::RPT + i, kc, ks_, kd_, mp.ck));
        vr[i] = ld16(row_ptr(r0 + mp.rgv * T::RPT + i, vc, vs_, vd_, mp.cv));
      }
    }
  };
  auto no_hook = [](int, const u32x4 (&)[T::RPT], const u32x4 (&)[T::RPT]) {};
  kv_sweep<D>(Ks, Vt, t_begin, t_end, mp, load, no_hook, [&](int t, const uint16_t* ks, const uint16_t* vt) {
    if (!wave_active) return;
    const int kv_valid = min(T::BN, L_kv - t * T::BN);
    tile_step<D, false>(st, ks, vt, l32, grp, p.scale_log2, kv_valid, 0, 0);
  });
  if (!wave_active || rho >= GL) return;

  const float ltot = st.l + __shfl_xor(st.l, 32);
  const float inv = 1.0f / ltot;
  const float lse2 = st.m + __log2f(ltot);
  if (p.S == 1) {
    const size_t orow = (((size_t)b * p.Ld + rr) * p.Hq + hq) * D;
    if (p.out_f32) store_row_f32<D>(reinterpret_cast<float*>(p.o_dec) + orow, st, inv, grp);
    else store_row_bf16<D>(reinterpret_cast<uint16_t*>(p.o_dec) + orow, st, inv, grp);
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
