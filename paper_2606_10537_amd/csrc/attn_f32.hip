// fp32 attention kernels (stage a prefill, Eq. 5 first sum, stage c decode).
//
// On MI355X the fp32 matrix-core peak equals the fp32 vector peak, so the fp32
// path runs on plain VALU FMAs: one thread owns one query row (q and the
// running output in registers), K/V tiles of 32 rows are staged in LDS and read
// by broadcast.  Probabilities stay fp32 throughout.
#include "pd_common.h"
#include "pd_kernels.h"

namespace pd {

constexpr int kF32Rows = 64;   // query rows per workgroup (one wave)
constexpr int kF32Keys = 32;   // keys per LDS tile

__device__ __forceinline__ f32x4 ld4(const float* p) { return *reinterpret_cast<const f32x4*>(p); }

template <int D>
struct RowState {
  float q[D], o[D];
  float m, l, qmass;
};

template <int D>
__device__ __forceinline__ void row_init(RowState<D>& st, const float* src) {
#pragma unroll
  for (int i = 0; i < D; i += 4) {
    f32x4 v = src ? ld4(src + i) : f32x4{0.f, 0.f, 0.f, 0.f};
    st.q[i] = v[0]; st.q[i + 1] = v[1]; st.q[i + 2] = v[2]; st.q[i + 3] = v[3];
  }
#pragma unroll
  for (int i = 0; i < D; ++i) st.o[i] = 0.f;
  st.m = -INFINITY;
  st.l = 0.f;
  st.qmass = 0.f;
}

// One LDS tile of `nk` valid keys; keys [qlo, qhi) (tile-relative) add to qmass.
template <int D>
__device__ __forceinline__ void row_tile(RowState<D>& st, const float (*Ks)[D], const float (*Vs)[D], int nk,
                                         float scale_log2, int qlo, int qhi) {
  float s[kF32Keys];
  float mt = -INFINITY;
#pragma unroll
  for (int kk = 0; kk < kF32Keys; ++kk) {
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < D; ++i) acc = fmaf(st.q[i], Ks[kk][i], acc);
    s[kk] = kk < nk ? acc * scale_log2 : -INFINITY;
    mt = fmaxf(mt, s[kk]);
  }
  if (mt > st.m) {
    const float a = fast_exp2(st.m - mt);
    st.m = mt;
    st.l *= a;
    st.qmass *= a;
#pragma unroll
    for (int i = 0; i < D; ++i) st.o[i] *= a;
  }
#pragma unroll
  for (int kk = 0; kk < kF32Keys; ++kk) {
    const float pv = fast_exp2(s[kk] - st.m);
    st.l += pv;
    if (kk >= qlo && kk < qhi) st.qmass += pv;
#pragma unroll
    for (int i = 0; i < D; ++i) st.o[i] = fmaf(pv, Vs[kk][i], st.o[i]);
  }
}

template <int D>
__device__ __forceinline__ void row_store(float* dst, const RowState<D>& st, float inv) {
#pragma unroll
  for (int i = 0; i < D; i += 4) {
    f32x4 v = {st.o[i] * inv, st.o[i + 1] * inv, st.o[i + 2] * inv, st.o[i + 3] * inv};
    *reinterpret_cast<f32x4*>(dst + i) = v;
  }
}

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void prefill_f32_kernel(PrefillArgs p) {
  __shared__ __attribute__((aligned(16))) float Ks[kF32Keys][D];
  __shared__ __attribute__((aligned(16))) float Vs[kF32Keys][D];
  const float* q_pre = reinterpret_cast<const float*>(p.q_pre);
  const float* k_pre = reinterpret_cast<const float*>(p.k_pre);
  const float* v_pre = reinterpret_cast<const float*>(p.v_pre);
  const float* q_qm = reinterpret_cast<const float*>(p.q_qm);
  const float* k_qm = reinterpret_cast<const float*>(p.k_qm);
  const float* v_qm = reinterpret_cast<const float*>(p.v_qm);
  float* o = reinterpret_cast<float*>(p.o);

  int lid = blockIdx.x;
  const int rb = lid % p.n_qt;
  lid /= p.n_qt;
  const int h = lid % p.Hq;
  lid /= p.Hq;
  const int n = lid % p.N;
  const int b = lid / p.N;
  const int g = h / p.G;
  const int C1 = p.C + 1;
  const size_t chunk = (size_t)b * p.N + n;
  const size_t qm_base = (p.qm_per_chunk ? chunk : (size_t)b) * (size_t)(p.Lq + p.Lm);
  const int tid = threadIdx.x;
  const int row = rb * kF32Rows + tid;

  RowState<D> st;
  const float* qsrc = nullptr;
  if (row < C1) qsrc = q_pre + ((chunk * C1 + row) * p.Hq + h) * D;
  else if (row < p.Sc) qsrc = q_qm + ((qm_base + (row - C1)) * p.Hq + h) * D;
  row_init<D>(st, qsrc);

  // Keys counted into qmass: the query columns for the BOS and content rows
  // (second sum of Eq. 5), the content columns for the query and pseudo-label
  // rows when the chunk score is asked for.
  const int qc_lo = C1, qc_hi = C1 + p.Lq;
  const int m_lo = row < C1 ? qc_lo : 1;
  const int m_hi = row < C1 ? qc_hi : (p.qm_mass ? C1 : 1);
  const int ntile = (p.Sc + kF32Keys - 1) / kF32Keys;
  constexpr int CPR = D / 4;
  for (int t = 0; t < ntile; ++t) {
    for (int i = tid; i < kF32Keys * CPR; i += kF32Rows) {
      const int kk = i / CPR, c = i % CPR;
      const int r = t * kF32Keys + kk;
      f32x4 kv = {0.f, 0.f, 0.f, 0.f}, vv = kv;
      if (r < C1) {
        const size_t off = ((chunk * C1 + r) * p.Hkv + g) * D + 4 * c;
        kv = ld4(k_pre + off);
        vv = ld4(v_pre + off);
      } else if (r < p.Sc) {
        const size_t off = ((qm_base + (r - C1)) * p.Hkv + g) * D + 4 * c;
        kv = ld4(k_qm + off);
        vv = ld4(v_qm + off);
      }
      *reinterpret_cast<f32x4*>(&Ks[kk][4 * c]) = kv;
      *reinterpret_cast<f32x4*>(&Vs[kk][4 * c]) = vv;
    }
    __syncthreads();
    const int t0 = t * kF32Keys;
    row_tile<D>(st, Ks, Vs, min(kF32Keys, p.Sc - t0), p.scale_log2, m_lo - t0, m_hi - t0);
    __syncthreads();
  }
  if (row >= p.Sc) return;
  const float inv = 1.0f / st.l;
  row_store<D>(o + ((chunk * p.Sc + row) * p.Hq + h) * D, st, inv);
  const size_t hb = chunk * p.Hq + h;
  if (row >= 1 && row < C1) p.part_i[hb * p.C + (row - 1)] = st.qmass * inv;
  if (row >= qc_lo && row < qc_hi) p.lse_q[hb * p.Lq + (row - qc_lo)] = st.m + __log2f(st.l);
  if (p.qm_mass && row >= C1) p.qm_mass[hb * (p.Lq + p.Lm) + (row - C1)] = st.qmass * inv;
}

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void escore_f32_kernel(EscoreArgs p) {
  __shared__ __attribute__((aligned(16))) float Qs[kF32Keys][D];
  __shared__ float Ls[kF32Keys];
  const float* q_qm = reinterpret_cast<const float*>(p.q_qm);
  const float* k_cache = reinterpret_cast<const float*>(p.k_cache);
  int lid = blockIdx.x;
  const int cb = lid % p.n_cb;
  lid /= p.n_cb;
  const int n = lid % p.N;
  const int b = lid / p.N;
  const int C1 = p.C + 1;
  const size_t chunk = (size_t)b * p.N + n;
  const size_t qm_base = (p.qm_per_chunk ? chunk : (size_t)b) * (size_t)(p.Lq + p.Lm);
  const int tid = threadIdx.x;
  const int j = cb * kF32Rows + tid;
  constexpr int CPR = D / 4;

  float acc = 0.f;
  for (int h = 0; h < p.Hq; ++h) {
    const int g = h / p.G;
    float kr[D];
    const float* ksrc = j < p.C ? k_cache + ((chunk * p.Hkv + g) * C1 + 1 + j) * D : nullptr;
#pragma unroll
    for (int i = 0; i < D; i += 4) {
      f32x4 v = ksrc ? ld4(ksrc + i) : f32x4{0.f, 0.f, 0.f, 0.f};
      kr[i] = v[0]; kr[i + 1] = v[1]; kr[i + 2] = v[2]; kr[i + 3] = v[3];
    }
    const float* lse = p.lse_q + (chunk * p.Hq + h) * p.Lq;
    for (int q0 = 0; q0 < p.Lq; q0 += kF32Keys) {
      for (int i = tid; i < kF32Keys * CPR; i += kF32Rows) {
        const int kk = i / CPR, c = i % CPR;
        const int r = q0 + kk;
        f32x4 v = {0.f, 0.f, 0.f, 0.f};
        if (r < p.Lq) v = ld4(q_qm + ((qm_base + r) * p.Hq + h) * D + 4 * c);
        *reinterpret_cast<f32x4*>(&Qs[kk][4 * c]) = v;
      }
      if (tid < kF32Keys) Ls[tid] = q0 + tid < p.Lq ? lse[q0 + tid] : INFINITY;
      __syncthreads();
      for (int kk = 0; kk < kF32Keys; ++kk) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < D; ++i) s = fmaf(Qs[kk][i], kr[i], s);
        acc += fast_exp2(s * p.scale_log2 - Ls[kk]);
      }
      __syncthreads();
    }
  }
  if (j < p.C) {
    float e = 0.f;
    if (!p.q2c)
      for (int h = 0; h < p.Hq; ++h) e += p.part_i[(chunk * p.Hq + h) * p.C + j];
    p.tok_score[chunk * p.C + j] = e + acc;
  }
}

// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void decode_f32_kernel(DecodeArgs p) {
  __shared__ __attribute__((aligned(16))) float Ks[kF32Keys][D];
  __shared__ __attribute__((aligned(16))) float Vs[kF32Keys][D];
  const float* q_dec = reinterpret_cast<const float*>(p.q_dec);
  const float* k_dec = reinterpret_cast<const float*>(p.k_dec);
  const float* v_dec = reinterpret_cast<const float*>(p.v_dec);
  const float* k_cache = reinterpret_cast<const float*>(p.k_cache);
  const float* v_cache = reinterpret_cast<const float*>(p.v_cache);
  const float* k_static = reinterpret_cast<const float*>(p.k_static);
  const float* v_static = reinterpret_cast<const float*>(p.v_static);

  int lid = blockIdx.x;
  const int sp = lid % p.S;
  lid /= p.S;
  const int rb = lid % p.n_qt;
  lid /= p.n_qt;
  const int h = lid % p.Hq;
  const int b = lid / p.Hq;
  const int g = h / p.G;
  const int C1 = p.C + 1;
  const int n_sel = p.n_sel;
  const int L_kv = n_sel + p.n_static + p.Ld;
  const int tid = threadIdx.x;
  const int r = rb * kF32Rows + tid;

  RowState<D> st;
  row_init<D>(st, r < p.Ld ? q_dec + (((size_t)b * p.Ld + r) * p.Hq + h) * D : nullptr);

  const int ntile = (L_kv + kF32Keys - 1) / kF32Keys;
  const int t_begin = (int)(((long long)ntile * sp) / p.S);
  const int t_end = (int)(((long long)ntile * (sp + 1)) / p.S);
  const size_t cache_bg = ((size_t)b * p.N * p.Hkv + g) * C1;
  const int32_t* cidx = p.chunk_idx + (size_t)b * p.K;
  const int32_t* tslot = p.tok_slot + (size_t)b * p.K * p.Bt;
  constexpr int CPR = D / 4;
  __shared__ int bad_index;   // checking build: some kept row of this shard was out of range
  if (kCheckIndices && tid == 0) bad_index = 0;
  if (kCheckIndices) __syncthreads();
  for (int t = t_begin; t < t_end; ++t) {
    for (int i = tid; i < kF32Keys * CPR; i += kF32Rows) {
      const int kk = i / CPR, c = i % CPR;
      const int j = t * kF32Keys + kk;
      f32x4 kv = {0.f, 0.f, 0.f, 0.f}, vv = kv;
      if (j < n_sel && p.compact) {
        const size_t off = ((((size_t)b * p.Hkv + g) * n_sel) + j) * D + 4 * c;
        kv = ld4(k_cache + off);
        vv = ld4(v_cache + off);
      } else if (j < n_sel) {
        const int q = j / (1 + p.Bt), s = j - q * (1 + p.Bt);
        int slot = s == 0 ? 0 : tslot[q * p.Bt + s - 1];
        int chunk = cidx[q];
        if (kCheckIndices && !kept_row_ok(chunk, slot, s == 0, p.N, p.C)) {
          chunk = 0;
          slot = 0;
          bad_index = 1;
        }
        const size_t off = (cache_bg + (size_t)chunk * p.Hkv * C1 + slot) * D + 4 * c;
        kv = ld4(k_cache + off);
        vv = ld4(v_cache + off);
      } else if (j < n_sel + p.n_static) {
        const size_t off = (((size_t)b * p.Ls + (j - n_sel)) * p.Hkv + g) * D + 4 * c;
        kv = ld4(k_static + off);
        vv = ld4(v_static + off);
      } else if (j < L_kv) {
        const size_t off = (((size_t)b * p.Ld + (j - n_sel - p.n_static)) * p.Hkv + g) * D + 4 * c;
        kv = ld4(k_dec + off);
        vv = ld4(v_dec + off);
      }
      *reinterpret_cast<f32x4*>(&Ks[kk][4 * c]) = kv;
      *reinterpret_cast<f32x4*>(&Vs[kk][4 * c]) = vv;
    }
    __syncthreads();
    row_tile<D>(st, Ks, Vs, min(kF32Keys, L_kv - t * kF32Keys), p.scale_log2, 0, 0);
    __syncthreads();
  }
  if (r >= p.Ld) return;
  float inv = 1.0f / st.l;
  float lse2 = st.m + __log2f(st.l);
  if (kCheckIndices && bad_index) inv = lse2 = __uint_as_float(kNanWord);
  if (p.S == 1) {
    row_store<D>(reinterpret_cast<float*>(p.o_dec) + (((size_t)b * p.Ld + r) * p.Hq + h) * D, st, inv);
    if (p.lse_dec) p.lse_dec[((size_t)b * p.Hq + h) * p.Ld + r] = lse2 * kLn2;
  } else {
    const size_t row = (((size_t)sp * p.B + b) * p.Hq + h) * p.Ld + r;
    row_store<D>(p.o_part + row * D, st, inv);
    p.lse_part[row] = lse2;
  }
}

// ---------------------------------------------------------------------------
template <int D>
static hipError_t prefill_f32_d(const PrefillArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(prefill_f32_kernel<D>, dim3(a.total), dim3(kF32Rows), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_prefill_f32(const PrefillArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? prefill_f32_d<128>(a, s) : prefill_f32_d<64>(a, s);
}

template <int D>
static hipError_t escore_f32_d(const EscoreArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(escore_f32_kernel<D>, dim3(a.total), dim3(kF32Rows), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_escore_f32(const EscoreArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? escore_f32_d<128>(a, s) : escore_f32_d<64>(a, s);
}

template <int D>
static hipError_t decode_f32_d(const DecodeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(decode_f32_kernel<D>, dim3(a.total), dim3(kF32Rows), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_decode_f32(const DecodeArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? decode_f32_d<128>(a, s) : decode_f32_d<64>(a, s);
}

}  // namespace pd
