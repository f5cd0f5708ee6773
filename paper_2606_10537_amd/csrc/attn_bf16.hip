// bf16 attention kernels for gfx950: chunk prefill (stage a) and sparse decode
// attention (stage c).  Both run one tile engine:
//
//   * a workgroup = kBf16Waves waves (32 query rows each), d = 64 or 128;
//   * K/V tiles of 64 rows go from HBM straight into LDS with
//     global_load_lds_dwordx4 (no register staging), kBf16Stages tiles
//     resident: the next ones stream in while the oldest is multiplied;
//   * both tiles are stored in 64-byte chunk groups with an XOR swizzle
//     (tile_off), so that the K fragment reads (ds_read_b128) and the
//     transposing V reads (ds_read_b64_tr_b16) are free of bank conflicts and
//     every fragment address is a per-lane base plus an immediate offset;
//   * S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_32x32x16_bf16 with
//     fp32 accumulation; Q stays in registers for the whole sweep;
//   * online softmax in the log2 domain, lazy rescaling of the running output
//     (only when a row maximum grows by more than 2^8), P rounded to bf16.
//
// Computing S transposed makes the MFMA output layout (each lane: one query,
// 16 keys) directly usable as the B operand of the P*V product.  The matching
// V^T operand (each lane: one d column, 8 keys) is produced from row-major V
// by ds_read_b64_tr_b16: within a group of 16 lanes, lane j receives element
// m of the 4 elements read by lane 4m + j/4, element j % 4.  If lane k of the
// group points at V[key0 + k/4][d0 + 4(k%4)], lane j therefore receives
// V[key0 + m][d0 + j], m = 0..3: four consecutive keys of one column.
#include "pd_common.h"
#include "pd_kernels.h"

namespace pd {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
#define PD_LDS __attribute__((address_space(3)))

template <int D>
struct Tile {
  static constexpr int NW = kBf16Waves;      // waves per workgroup
  static constexpr int NH = kBf16RowsPerWave / 32;   // 32-row groups per wave
  static constexpr int BM = kBf16Rows;       // query rows per workgroup
  static constexpr int BN = 64;              // key rows per KV tile
  static constexpr int NT = 64 * NW;         // threads per workgroup
  static constexpr int S = kBf16Stages;      // resident K/V tiles
  static constexpr int CH = D / 8;           // 16-byte chunks per row
  static constexpr int BPW = CH / NW;        // 1 KB DMA blocks (16 rows x 64 B) per wave and tile, K and V
  static constexpr int KS = D / 16;          // MFMA k-steps along d
  static constexpr int DB = D / 32;          // 32-row blocks of O^T
  static constexpr int TILE = BN * D;        // elements of one K or V tile
  static_assert(BPW >= 1, "unsupported head dim");
};

// LDS layout of a 64-row K or V tile, in elements: logical 16-byte chunk c of
// row r sits at (c / 4) * 2048 + r * 32 + 8 * ((c % 4) ^ ((r / 4) % 4)), i.e.
// 64-byte chunk groups of all 64 rows one after the other, with the chunks of
// a group XOR-swizzled by bits 2-3 of the row.  LDS has 64 banks (256 bytes per
// bank row); ds_read_b128 serves 16 lanes per pass and ds_read_b64 32 lanes,
// and a pass is conflict-free when its lanes cover a whole bank row.  A K
// fragment pass reads one chunk of 16 consecutive rows (rows r % 4 and r / 4 %
// 4 pick 16 distinct 16-byte bank groups); a transposing V pass reads 4 chunks
// of 4 consecutive rows (again 16 distinct groups).  A 1 KB DMA block is 16
// rows of one chunk group.
__device__ __forceinline__ int tile_off(int r, int c) { return (c >> 2) * 2048 + r * 32 + 8 * ((c & 3) ^ ((r >> 2) & 3)); }

// Wave group of a wave (0 or 1): one wave of each group per SIMD.
#ifndef PD_GROUP_OF_WAVE
#define PD_GROUP_OF_WAVE(w) ((w) >> 2)
#endif
__device__ __forceinline__ int wave_group(int wave) {
  return (kBf16Waves == 8 && kBf16RowsPerWave == 32) ? PD_GROUP_OF_WAVE(wave) : 0;
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

__device__ __forceinline__ i16x4 ld_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((PD_LDS i16x4*)(p));
}

// 16 bytes from global memory into LDS slot `lane` of the 1 KB block at lds
// (global_load_lds_dwordx4 with the block's LDS address in M0).  Issued as
// inline assembly: when the compiler sees an LDS DMA in flight it can no longer
// count LDS reads precisely and waits for all of them (lgkmcnt(0)) before every
// fragment use.  Completion is tracked by hand (wait_dma_keep); loads the
// compiler does not see only make its own vmcnt waits stricter.
__device__ __forceinline__ void dma16(const uint16_t* g, uint16_t* lds) {
  const uint32_t lds_addr = (uint32_t)(uintptr_t)(PD_LDS void*)(lds);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_addr) : "memory", "m0");
}

// Engine state of 32 query rows of a wave (a wave holds NH of them).
template <int D>
struct WaveState {
  bf16x8 qf[Tile<D>::KS];
  f32x16 o[Tile<D>::DB];
  float m;      // running row max (log2 domain), shared by lanes l and l^32
  float l;      // this lane's partial sum of the bf16-rounded weights that multiply V
  float lx;     // this lane's partial sum of the unrounded weights (prefill only)
  float qmass;  // this lane's partial mass on its counted key range (prefill only)
};

// Keys counted into qmass (prefill only), tile-relative: a lane whose query row
// lies below `split` (row index within the wave's first row group; +32 per
// further group) counts [lo0, hi0), the other lanes [lo1, hi1).  The prefill
// counts the query columns for the BOS and content rows (Eq. 5, first sum)
// and the content columns for the query and pseudo-label rows (the
// prefill-time chunk score).
struct MassRange {
  int split, lo0, hi0, lo1, hi1;
};

// Lane-constant parts of the LDS fragment addresses (elements).  Everything
// else (k-step, key block, d block, tile buffer) is an immediate offset.
struct FragAddr {
  int k[2];   // K fragment, row l32 (+ 32 kb), chunk 2 ks + grp: base for ks % 2, + (ks / 2) * 2048 + kb * 1024
  int v[2];   // V transposing read: base for r2, + db * 2048 + (16 kk + 8 r2) * 32
  __device__ FragAddr(int lane) {
    const int l32 = lane & 31, grp = lane >> 5;
#pragma unroll
    for (int j = 0; j < 2; ++j) k[j] = tile_off(l32, 2 * j + grp);
    // Group q = lane / 16 of 16 lanes, kq = lane % 16: this lane points at
    // V[4 grp + kq/4 + 16 kk + 8 r2][32 db + 16 (q % 2) + 4 (kq % 4)], 4 elements.
    const int kq = lane & 15, dh = (lane >> 4) & 1;
    const int row = 4 * grp + (kq >> 2), c = 2 * dh + ((kq & 3) >> 1);
#pragma unroll
    for (int j = 0; j < 2; ++j) v[j] = tile_off(row + 8 * j, c) - 8 * 32 * j + 4 * (kq & 1);
  }
};

// One KV tile for one wave, in three phases: S^T = K Q^T (s_phase), online
// softmax producing the bf16 weights P (softmax_phase), O^T += V^T P^T
// (pv_phase).  kv_valid: number of valid keys in this tile (64 except in a
// ragged last tile).  mr: keys counted into qmass.  EXACT: also keep the
// unrounded row sum and the counted mass (prefill).  O is normalised by the sum of the same
// bf16-rounded weights that multiply V, so rounding P perturbs a convex
// combination instead of scaling O.
template <int D>
__device__ __forceinline__ bf16x8 k_frag(const uint16_t* Ks, const FragAddr& fa, int ks, int kb) {
  return __builtin_bit_cast(bf16x8, ld16(Ks + fa.k[ks & 1] + (ks >> 1) * 2048 + kb * 1024));
}

// Fragments are read PF k-steps ahead of the MFMAs that use them (kept in that
// order by scheduling fences); each K fragment serves the NH row groups.
#ifndef PD_S_PREFETCH
#define PD_S_PREFETCH 2
#endif
#ifndef PD_PIN_S
#define PD_PIN_S 1
#endif
template <int D, int NH>
__device__ __forceinline__ void s_phase(f32x16 (&s)[NH][2], const WaveState<D> (&st)[NH], const uint16_t* Ks,
                                        const FragAddr& fa) {
  using T = Tile<D>;
  constexpr int PF = PD_S_PREFETCH < T::KS ? PD_S_PREFETCH : T::KS - 1;
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) s[h][kb] = f32x16{0};
  bf16x8 a[PF + 1][2];
#pragma unroll
  for (int ks = 0; ks < PF; ++ks)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) a[ks][kb] = k_frag<D>(Ks, fa, ks, kb);
#pragma unroll
  for (int ks = 0; ks < T::KS; ++ks) {
    if (ks + PF < T::KS) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) a[(ks + PF) % (PF + 1)][kb] = k_frag<D>(Ks, fa, ks + PF, kb);
    }
    if (PD_PIN_S) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int h = 0; h < NH; ++h) s[h][kb] = mfma32x32x16(a[ks % (PF + 1)][kb], st[h].qf[ks], s[h][kb]);
    if (PD_PIN_S) __builtin_amdgcn_sched_barrier(0);
  }
}

// Max of this lane's value and the value of lane l ^ 32 (v_permlane32_swap
// exchanges the two halves of the wave without going through LDS).
__device__ __forceinline__ float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Softmax of one 32-row group, part 1: mask, row max, lazy rescale of the
// running output.  Returns -m (log2 domain) for the exponent FMA.  Key of
// s[kb][r]: 32*kb + 8*(r/4) + 4*grp + r%4.  The max is taken on raw scores (the
// scale is positive) and the scale is folded into one FMA: p = exp2(s * scale_log2 - m).
template <int D, bool EXACT>
__device__ __forceinline__ float softmax_max(WaveState<D>& st, f32x16 (&s)[2], int grp, float scale_log2,
                                             int kv_valid) {
  using T = Tile<D>;
  if (kv_valid < 64) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + 8 * (r >> 2) + 4 * grp + (r & 3);
        s[kb][r] = key < kv_valid ? s[kb][r] : -INFINITY;
      }
  }
  // One v_max3_f32 per pair (the file is built without NaN semantics, so no
  // canonicalising v_max precedes each score).
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; r += 2) mx = fmaxf(fmaxf(mx, s[kb][r]), s[kb][r + 1]);
  mx = max_across_halves(mx) * scale_log2;
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
  return -st.m;
}

// Part 2 (branch-free): weights p, packed to bf16 in pk; s keeps the fp32 p
// for the counted mass.  The rounded weights' sum goes into l (one
// v_dot2c_f32_bf16 with (1, 1) per packed pair), the exact sum into lx; the
// exact sum of this tile is returned.
template <int D, bool EXACT>
__device__ __forceinline__ float softmax_exp(WaveState<D>& st, f32x16 (&s)[2], uint32_t (&pk)[16], float nm,
                                             float scale_log2) {
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
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float lr = st.l;
#pragma unroll
  for (int i = 0; i < 16; ++i) lr = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[i]), ones, lr, false);
  st.l = lr;
  return lsum;
}

// Part 3 (prefill only): mass of this lane's counted keys (row group h of the
// wave).  A range covering the whole tile takes the tile's exact row sum; the
// per-key test runs only in tiles where some lane's range is partial.
template <int D>
__device__ __forceinline__ void softmax_qmass(WaveState<D>& st, const f32x16 (&s)[2], int grp, int h,
                                              const MassRange& mr, float lsum) {
  if (mr.lo0 >= mr.hi0 && mr.lo1 >= mr.hi1) return;   // wave-uniform: nothing counted in this tile
  const int l32 = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) & 31;   // lane % 32
  const bool first = l32 + 32 * h < mr.split;
  const int qlo = first ? mr.lo0 : mr.lo1, qhi = first ? mr.hi0 : mr.hi1;
  const bool any = qlo < qhi;
  float qs = lsum;
  if (__ballot(any && (qlo > 0 || qhi < 64))) {
    qs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + 8 * (r >> 2) + 4 * grp + (r & 3);
        qs += (key >= qlo && key < qhi) ? s[kb][r] : 0.f;
      }
  }
  st.qmass += any ? qs : 0.f;
}

template <int D, bool EXACT>
__device__ __forceinline__ void softmax_phase(WaveState<D>& st, f32x16 (&s)[2], uint32_t (&pk)[16], int grp, int h,
                                              float scale_log2, int kv_valid, const MassRange& mr) {
  const float nm = softmax_max<D, EXACT>(st, s, grp, scale_log2, kv_valid);
  const float lsum = softmax_exp<D, EXACT>(st, s, pk, nm, scale_log2);
  if constexpr (EXACT) softmax_qmass<D>(st, s, grp, h, mr, lsum);
}

// V^T fragment of k-step kk and d block db (two transposing reads).
template <int D>
__device__ __forceinline__ bf16x8 v_frag(const uint16_t* Vs, const FragAddr& fa, int kk, int db) {
  const uint16_t* vb = Vs + db * 2048 + 16 * kk * 32;
  const i16x4 lo = ld_tr16(vb + fa.v[0]);
  const i16x4 hi = ld_tr16(vb + fa.v[1] + 8 * 32);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// The first two V fragments of a tile's P*V (fragments i = 0, 1 below).
template <int D>
__device__ __forceinline__ void v_pre(bf16x8 (&vp)[2], const uint16_t* Vs, const FragAddr& fa) {
  using T = Tile<D>;
  vp[0] = v_frag<D>(Vs, fa, 0, 0);
  vp[1] = v_frag<D>(Vs, fa, 1 / T::DB, 1 % T::DB);
}

// P^T operand of k-step kk: keys 16kk + 4grp + {0..3} then 16kk + 8 + 4grp + {0..3}
// (pk[4kk .. 4kk+3]); the two transposing reads deliver V^T in that order.
// Fragments are read two MFMAs ahead (the first two, vp, by the caller); each
// serves the NH row groups.
template <int D, int NH>
__device__ __forceinline__ void pv_phase(WaveState<D> (&st)[NH], const uint32_t (&pk)[NH][16], const uint16_t* Vs,
                                         const FragAddr& fa, const bf16x8 (&vp)[2]) {
  using T = Tile<D>;
  constexpr int N = 4 * T::DB;   // fragments: i = kk * DB + db
  bf16x8 a[3];
  a[0] = vp[0];
  a[1] = vp[1];
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if (i + 2 < N) a[(i + 2) % 3] = v_frag<D>(Vs, fa, (i + 2) / T::DB, (i + 2) % T::DB);
    const int kk = i / T::DB, db = i % T::DB;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const bf16x8 pf =
          __builtin_bit_cast(bf16x8, u32x4{pk[h][4 * kk], pk[h][4 * kk + 1], pk[h][4 * kk + 2], pk[h][4 * kk + 3]});
      st[h].o[db] = mfma32x32x16(a[i % 3], pf, st[h].o[db]);
    }
  }
}

// The tile step of one wave.  With one row group per wave (two waves per
// SIMD), the two wave groups of a workgroup (one wave of each per SIMD) run the
// phases in different orders so that one group's softmax overlaps the other's
// MFMAs: group 0 does S, softmax, P*V of tile t; group 1 first does the P*V of
// tile t-1 (its weights are still in pk), then S and softmax of tile t, and the
// P*V of the last tile right after its softmax.  The order of the
// online-softmax updates is the same in both groups.  One code path with
// wave-uniform guards keeps a single pk array.  With two row groups per wave
// (one wave per SIMD) each K and V fragment serves both groups.  VPRE: the
// first two V fragments of the tile's P*V are read right after its S, so that
// they are in flight during the softmax (in group 1, until the next step)
// rather than at the start of the P*V; it shortens the prefill by about 2.6 %
// and lengthens the decode, whose register allocation it changes, by about as
// much, so only the prefill uses it.
template <int D, int NH, bool EXACT, bool VPRE>
__device__ __forceinline__ void wave_step(WaveState<D> (&st)[NH], uint32_t (&pk)[NH][16], bf16x8 (&vp)[2],
                                          bool deferred, bool first, bool last, const uint16_t* Ks,
                                          const uint16_t* Vs, const uint16_t* Vs_prev, const FragAddr& fa, int grp,
                                          float scale_log2, int kv_valid, const MassRange& mr) {
  f32x16 s[NH][2];
  if (deferred && !first) {
    if (!VPRE) v_pre<D>(vp, Vs_prev, fa);
    pv_phase<D, NH>(st, pk, Vs_prev, fa, vp);
  }
  s_phase<D, NH>(s, st, Ks, fa);
  if (VPRE) v_pre<D>(vp, Vs, fa);   // in flight during the softmax (and, deferred, until the next step)
#pragma unroll
  for (int h = 0; h < NH; ++h) softmax_phase<D, EXACT>(st[h], s[h], pk[h], grp, h, scale_log2, kv_valid, mr);
  if (!deferred || last) {
    if (!VPRE) v_pre<D>(vp, Vs, fa);
    pv_phase<D, NH>(st, pk, Vs, fa, vp);
  }
}

// Completes the loads of the Q fragments here, before the sweep.  The compiler
// does not see the tile DMAs (inline assembly): a Q load it still counted as
// pending would make it wait for every load in flight (s_waitcnt vmcnt(0)),
// tile DMAs included, at the fragment's first use in every tile.  Consuming
// the registers in an empty asm statement puts that one wait here instead.
template <int D, int NH>
__device__ __forceinline__ void q_landed(const WaveState<D> (&st)[NH]) {
#pragma unroll
  for (int j = 0; j < NH; ++j)
#pragma unroll
    for (int ks = 0; ks < Tile<D>::KS; ++ks) asm volatile("" ::"v"(st[j].qf[ks]));
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

// Global element pointers of one K row and one V row.
struct RowPtr {
  const uint16_t* k;
  const uint16_t* v;
};

// Issue this wave's share of the DMA of one K/V tile: BPW blocks for K and
// for V.  Block b holds rows 16 (b % 4) .. +15 of chunk group b / 4; lane
// takes row 16 (b % 4) + lane / 4 and loads the logical chunk that tile_off
// places in its 16-byte slot.  row(r) returns the global K and V pointers of
// tile row r (already clamped to a valid row).  All row pointers are formed
// before the first DMA is issued: an LDS read (a row table) after a DMA would
// make the compiler wait for it.
template <int D>
__device__ __forceinline__ int dma_row(int wave, int lane, int j) {
  return ((wave * Tile<D>::BPW + j) & 3) * 16 + (lane >> 2);
}

template <int D>
__device__ __forceinline__ void dma_tile_rows(uint16_t* Kd, uint16_t* Vd, int wave, int lane,
                                              const RowPtr (&rp)[Tile<D>::BPW]) {
  using T = Tile<D>;
#pragma unroll
  for (int j = 0; j < T::BPW; ++j) {
    const int blk = wave * T::BPW + j;
    const int r = dma_row<D>(wave, lane, j);
    const int c = 4 * (blk >> 2) + ((lane & 3) ^ ((r >> 2) & 3));
    dma16(rp[j].k + 8 * c, Kd + blk * 512);
    dma16(rp[j].v + 8 * c, Vd + blk * 512);
  }
}

template <int D, class Row>
__device__ __forceinline__ void dma_tile(uint16_t* Kd, uint16_t* Vd, int wave, int lane, Row&& row) {
  RowPtr rp[Tile<D>::BPW];
#pragma unroll
  for (int j = 0; j < Tile<D>::BPW; ++j) rp[j] = row(dma_row<D>(wave, lane, j));
  dma_tile_rows<D>(Kd, Vd, wave, lane, rp);
}

// Wait until this wave has at most `newer` tiles of DMA in flight: tile DMAs
// are loads and complete in issue order, so the tile issued before those has
// landed (stores issued in between can only make the wait longer).
template <int PER>
__device__ __forceinline__ void wait_dma_keep(int newer) {
  if (newer <= 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if (newer == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(PER) : "memory");
  else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * PER) : "memory");
}

// Workgroup barrier without a memory fence.  __syncthreads() would also wait
// for every LDS DMA still in flight (they count as outstanding LDS writes),
// draining the pipeline; here the tile in use is covered by wait_dma_keep, and
// every LDS read of older tiles has been consumed before a wave gets here.  The
// memory clobber keeps the compiler from moving memory accesses across it.
__device__ __forceinline__ void tile_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Pipelined sweep over KV tiles [t_begin, t_end) with S resident tiles: tile t
// lives in buffer (t - t_begin) % S.  When tile t is computed, tile t-1 is still
// resident (its V feeds the deferred P*V of wave group 1), t+1 .. t+PF-1 are in
// flight and t+PF (PF = S-2) is issued into the buffer of tile t-2.  One
// barrier per tile: after it, tile t has landed for every wave and every wave
// is done with tile t-1's step.  The buffers are distinct LDS objects and every
// buffer index is a compile-time constant (the loop is unrolled by S), so the
// compiler never mistakes a DMA into one buffer for a write to another.
// dma(t, Kd, Vd) issues a tile, hook(t, Ks, Vs) sees a landed tile (the prefill
// writes its cache share there), step(t, Ks, Vs, Vs_prev, last) computes.
template <int D, class Dma, class Hook, class Step>
__device__ __forceinline__ void kv_sweep(uint16_t* const* Kb, uint16_t* const* Vb, int t_begin, int t_end,
                                         Dma&& dma, Hook&& hook, Step&& step) {
  constexpr int S = Tile<D>::S, PF = S - 2, PER = 2 * Tile<D>::BPW;
#pragma unroll
  for (int i = 0; i < PF; ++i)
    if (t_begin + i < t_end) dma(t_begin + i, Kb[i], Vb[i]);
  for (int t = t_begin; t < t_end; t += S) {
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const int tt = t + i;
      if (tt < t_end) {
        wait_dma_keep<PER>(min(PF - 1, t_end - 1 - tt));
        tile_barrier();
        if (tt + PF < t_end) dma(tt + PF, Kb[(i + PF) % S], Vb[(i + PF) % S]);
        hook(tt, Kb[i], Vb[i]);
        step(tt, Kb[i], Vb[i], Vb[(i + S - 1) % S], tt == t_end - 1);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Stage (a): chunk prefill.  Workgroup = (b, n, h, 256-row query tile).
// Also writes the chunk KV cache (each KV tile by exactly one workgroup of the
// (b, n, kv-head) group), the per-head query-column mass of the content rows,
// the log2-domain LSE of the query rows and, when asked, the per-head
// content mass of the query and pseudo-label rows.
template <int D>
__global__ __launch_bounds__(Tile<D>::NT, 1) void prefill_bf16_kernel(PrefillArgs p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t K0[T::TILE], K1[T::TILE], K2[T::TILE], K3[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t V0[T::TILE], V1[T::TILE], V2[T::TILE], V3[T::TILE];
  __shared__ __attribute__((aligned(16))) float kacc[T::NT / T::CH * D];   // content-key sums, one slot per thread
  uint16_t* const Kb[4] = {K0, K1, K2, K3};   // the first T::S are used
  uint16_t* const Vb[4] = {V0, V1, V2, V3};

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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

  // Q fragments of this lane's query rows (one per row group j).
  WaveState<D> st[T::NH];
  const bool wave_active = qt * T::BM + wave * T::NH * 32 < p.Sc;
#pragma unroll
  for (int j = 0; j < T::NH; ++j) {
    const int qrow = qt * T::BM + (wave * T::NH + j) * 32 + l32;
    const uint16_t* src = nullptr;
    if (qrow < C1) src = p.q_pre + ((chunk * C1 + qrow) * p.Hq + h) * D;
    else if (qrow < p.Sc) src = p.q_qm + ((qm_base + (qrow - C1)) * p.Hq + h) * D;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks)
      st[j].qf[ks] = src ? __builtin_bit_cast(bf16x8, ld16(src + 16 * ks + 8 * grp)) : bf16x8{0};
    wave_init(st[j]);
  }
  q_landed<D, T::NH>(st);
  const FragAddr fa(lane);

  // Row r of the chunk sequence lives at base + r*HD (HD = H_kv*d elements), with
  // base the chunk's rows for r <= C and the shared query/pseudo-label rows after.
  // Rows past the end are clamped to the last row: their keys are masked out of
  // the softmax and their (finite) values get probability 0.
  const int HD = p.Hkv * D;
  const uint16_t* k_lo = p.k_pre + (chunk * C1 * p.Hkv + g) * D;
  const uint16_t* v_lo = p.v_pre + (chunk * C1 * p.Hkv + g) * D;
  const uint16_t* k_hi = p.k_qm + (qm_base * p.Hkv + g) * D - (size_t)C1 * HD;
  const uint16_t* v_hi = p.v_qm + (qm_base * p.Hkv + g) * D - (size_t)C1 * HD;
  auto dma = [&](int t, uint16_t* Kd, uint16_t* Vd) {
    const int r0 = t * T::BN;
    dma_tile<D>(Kd, Vd, wave, lane, [=](int r) {
      const int rr = min(r0 + r, p.Sc - 1);
      const bool lo = rr < C1;
      const unsigned off = (unsigned)rr * HD;
      return RowPtr{(lo ? k_lo : k_hi) + off, (lo ? v_lo : v_hi) + off};
    });
  };
  // Each KV tile of the (b, n, kv head) group is written to the cache by exactly
  // one workgroup of that group (query tile t % n_qt of head g*G + (t / n_qt) % G),
  // from the landed LDS tile: thread tid copies logical chunks tid + NT i.
  // Thread tid always handles 16-byte chunk tid % CH of the rows it copies, so
  // its content-key sums live in its own LDS slot kacc[tid / CH][8 (tid % CH) ..]
  // (no other thread touches it until the reduction after the sweep).
  float* const kslot = kacc + (tid / T::CH) * D + 8 * (tid % T::CH);
#pragma unroll
  for (int e = 0; e < 8; ++e) kslot[e] = 0.f;
  auto cache_write = [&](int t, const uint16_t* Ks, const uint16_t* Vs) {
    const bool writer = (t % p.n_qt == qt) && ((t / p.n_qt) % p.G == h % p.G);
    if (!writer) return;
    const size_t base = (chunk * p.Hkv + g) * C1;
    float ksum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < T::BN * T::CH / T::NT; ++i) {
      const int u = tid + T::NT * i;
      const int r = u / T::CH, c = u % T::CH;
      const int row = t * T::BN + r;
      if (row < C1) {
        const u32x4 kv = ld16(Ks + tile_off(r, c));
        st16(p.k_cache + (base + row) * D + 8 * c, kv);
        st16(p.v_cache + (base + row) * D + 8 * c, ld16(Vs + tile_off(r, c)));
        if (row >= 1) {   // content rows only (the BOS row is not part of the key mean)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            ksum[2 * q] += __uint_as_float(kv[q] << 16);
            ksum[2 * q + 1] += __uint_as_float(kv[q] & 0xffff0000u);
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) kslot[e] += ksum[e];
  };

  const int qc_lo = C1, qc_hi = C1 + p.Lq;   // query columns counted by Eq. 5
  const int cm_hi = p.qm_mass ? C1 : 1;       // content columns counted for the chunk score (if asked)
  const int split = C1 - (qt * T::BM + wave * T::NH * 32);
  uint32_t pk_prev[T::NH][16];
  bf16x8 vp_prev[2];
  const bool deferred = wave_group(wave) != 0;
  kv_sweep<D>(Kb, Vb, 0, p.n_kvt, dma, cache_write,
              [&](int t, const uint16_t* ks, const uint16_t* vs, const uint16_t* vs_prev, bool last) {
                if (!wave_active) return;
                const int t0 = t * T::BN;
                const int kv_valid = min(T::BN, p.Sc - t0);
                const MassRange mr{split, max(qc_lo - t0, 0), min(qc_hi - t0, T::BN), max(1 - t0, 0),
                                   min(cm_hi - t0, T::BN)};
                wave_step<D, T::NH, true, true>(st, pk_prev, vp_prev, deferred, t == 0, last, ks, vs, vs_prev, fa,
                                                grp, p.scale_log2, kv_valid, mr);
              });
  // This workgroup's content-key sums: the thread slots summed in a fixed
  // order, one vector per (b, n, kv head, writer slot qt*G + h%G).
  __syncthreads();
  if (tid < D) {
    float sum = 0.f;
    for (int r = 0; r < T::NT / T::CH; ++r) sum += kacc[r * D + tid];
    p.km_part[((chunk * p.Hkv + g) * (size_t)(p.n_qt * p.G) + qt * p.G + h % p.G) * D + tid] = sum;
  }
  if (!wave_active) return;

#pragma unroll
  for (int j = 0; j < T::NH; ++j) {
    const int qrow = qt * T::BM + (wave * T::NH + j) * 32 + l32;
    const float ltot = st[j].l + __shfl_xor(st[j].l, 32);
    const float lxtot = st[j].lx + __shfl_xor(st[j].lx, 32);
    const float qtot = st[j].qmass + __shfl_xor(st[j].qmass, 32);
    const float inv = 1.0f / ltot;
    if (qrow < p.Sc) {
      const size_t orow = ((chunk * p.Sc + qrow) * p.Hq + h) * D;
      if (p.out_f32) store_row_f32<D>(reinterpret_cast<float*>(p.o) + orow, st[j], inv, grp);
      else store_row_bf16<D>(p.o + orow, st[j], inv, grp);
      if (grp == 0) {
        const size_t hb = chunk * p.Hq + h;
        if (qrow >= 1 && qrow < C1) p.part_i[hb * p.C + (qrow - 1)] = qtot / lxtot;
        if (qrow >= qc_lo && qrow < qc_hi) p.lse_q[hb * p.Lq + (qrow - qc_lo)] = st[j].m + __log2f(lxtot);
        if (p.qm_mass && qrow >= C1) p.qm_mass[hb * (p.Lq + p.Lm) + (qrow - C1)] = qtot / lxtot;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Stage (c): sparse decode attention.  Workgroup = (b, kv head g, 128-row tile
// of the G*L_d query rows of that group, KV shard).  Query row rho of the group
// is head g*G + rho / L_d, decode row rho % L_d.  KV row j of the shard walks:
// [kept chunks: BOS + kept slots] ; [static rows] ; [own rows].
template <int D>
__global__ __launch_bounds__(Tile<D>::NT, 1) void decode_bf16_kernel(DecodeArgs p) {
  using T = Tile<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t K0[T::TILE], K1[T::TILE], K2[T::TILE], K3[T::TILE];
  __shared__ __attribute__((aligned(1024))) uint16_t V0[T::TILE], V1[T::TILE], V2[T::TILE], V3[T::TILE];
  uint16_t* const Kb[4] = {K0, K1, K2, K3};   // the first T::S are used
  uint16_t* const Vb[4] = {V0, V1, V2, V3};
  __shared__ __attribute__((aligned(16))) int rowtab[kDecodeTableRows];   // cache row (n*Hkv*(C+1) + slot) of gathered rows

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  const int n_sel = p.n_sel;
  const int L_kv = n_sel + p.n_static + p.Ld;

  WaveState<D> st[T::NH];
  const bool wave_active = qt * T::BM + wave * T::NH * 32 < GL;
#pragma unroll
  for (int j = 0; j < T::NH; ++j) {
    const int rho = qt * T::BM + (wave * T::NH + j) * 32 + l32;
    const int hq = g * p.G + (rho < GL ? rho / p.Ld : 0);
    const int rr = rho < GL ? rho % p.Ld : 0;
    const uint16_t* src = rho < GL ? p.q_dec + (((size_t)b * p.Ld + rr) * p.Hq + hq) * D : nullptr;
#pragma unroll
    for (int ks = 0; ks < T::KS; ++ks)
      st[j].qf[ks] = src ? __builtin_bit_cast(bf16x8, ld16(src + 16 * ks + 8 * grp)) : bf16x8{0};
    wave_init(st[j]);
  }
  const FragAddr fa(lane);

  // This shard's tiles.
  const int n_kvt = (L_kv + T::BN - 1) / T::BN;
  const int t_begin = (int)(((long long)n_kvt * sp) / p.S);
  const int t_end = (int)(((long long)n_kvt * (sp + 1)) / p.S);

  // Prefix rows of (b, g): gathered from the chunk cache (row n*Hkv*C1 + slot
  // from this base), or, in compact mode, row j of the contiguous buffer.
  const size_t cache_bg = p.compact ? ((size_t)b * p.Hkv + g) * n_sel : ((size_t)b * p.N * p.Hkv + g) * C1;
  // Prefix rows of this shard: row codes into LDS once (the host keeps every
  // shard within kDecodeTableRows rows), so tile loads need no index fetch.
  const int j_lo = t_begin * T::BN;
  const int j_hi = min(t_end * T::BN, n_sel);
  __shared__ int bad_index;   // checking build: some kept row of this shard was out of range
  if (kCheckIndices && tid == 0) bad_index = 0;
  if (kCheckIndices) __syncthreads();
  if (p.compact) {
    for (int j = j_lo + tid; j < j_hi; j += T::NT) rowtab[j - j_lo] = j;
  } else {
    const int32_t* cidx = p.chunk_idx + (size_t)b * p.K;
    const int32_t* tslot = p.tok_slot + (size_t)b * p.K * p.Bt;
    for (int j = j_lo + tid; j < j_hi; j += T::NT) {
      const int kk = j / (1 + p.Bt), s = j - kk * (1 + p.Bt);
      int slot = s == 0 ? 0 : tslot[kk * p.Bt + s - 1];
      int chunk = cidx[kk];
      if (kCheckIndices && !kept_row_ok(chunk, slot, s == 0, p.N, p.C)) {
        chunk = 0;
        slot = 0;
        bad_index = 1;
      }
      rowtab[j - j_lo] = chunk * p.Hkv * C1 + slot;
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
  const int n_static = p.n_static;
  int* const rowtab_p = rowtab;
  // A whole gathered tile takes this lane's row codes from the row table.
  // They are read one tile ahead (right after the previous tile's DMA) and
  // kept raw until used, so that issuing a DMA after the barrier needs no LDS
  // read and no wait.
  auto read_tab = [=](int t, unsigned (&o)[T::BPW]) {
    const int* tab = rowtab_p + (t * T::BN - j_lo);
#pragma unroll
    for (int j = 0; j < T::BPW; ++j) o[j] = (unsigned)tab[dma_row<D>(wave, lane, j)];
  };
  unsigned nxt[T::BPW];
  int nxt_t = -1;
  auto dma = [&](int t, uint16_t* Kd, uint16_t* Vd) {
    const int* rowtab = rowtab_p;
    const int r0 = t * T::BN;
    if (r0 + T::BN <= n_sel) {
      // Whole tile gathered from the cache.
      unsigned o[T::BPW];
      if (nxt_t == t) {
#pragma unroll
        for (int j = 0; j < T::BPW; ++j) o[j] = nxt[j];
      } else {
        read_tab(t, o);
      }
      RowPtr rp[T::BPW];
#pragma unroll
      for (int j = 0; j < T::BPW; ++j) rp[j] = RowPtr{kc + o[j] * D, vc + o[j] * D};
      dma_tile_rows<D>(Kd, Vd, wave, lane, rp);
      if (r0 + 2 * T::BN <= n_sel && t + 1 < t_end) {
        read_tab(t + 1, nxt);
        nxt_t = t + 1;
      }
    } else if (r0 >= n_sel) {
      // No gathered row: static rows, then own rows.
      dma_tile<D>(Kd, Vd, wave, lane, [=](int r) {
        const int j = min(r0 + r, L_kv - 1);
        const unsigned off = (unsigned)(j * HD);
        const bool stat = j < n_sel + n_static;
        return RowPtr{(stat ? ks_ : kd_) + off, (stat ? vs_ : vd_) + off};
      });
    } else {
      dma_tile<D>(Kd, Vd, wave, lane, [=](int r) {
        const int j = min(r0 + r, L_kv - 1);
        const unsigned tab = (unsigned)rowtab[min(max(j - j_lo, 0), tab_hi)] * D;
        const bool gath = j < n_sel, stat = j < n_sel + n_static;
        const unsigned off = gath ? tab : (unsigned)(j * HD);
        const uint16_t* kb = stat ? ks_ : kd_;
        const uint16_t* vb = stat ? vs_ : vd_;
        kb = gath ? kc : kb;
        vb = gath ? vc : vb;
        return RowPtr{kb + off, vb + off};
      });
    }
  };
  // The Q loads overlap the row-table loads above; both have landed here.
  q_landed<D, T::NH>(st);
  auto no_hook = [](int, const uint16_t*, const uint16_t*) {};
  uint32_t pk_prev[T::NH][16];
  bf16x8 vp_prev[2];
  const bool deferred = wave_group(wave) != 0;
  kv_sweep<D>(Kb, Vb, t_begin, t_end, dma, no_hook,
              [&](int t, const uint16_t* ks, const uint16_t* vs, const uint16_t* vs_prev, bool last) {
                if (!wave_active) return;
                const int kv_valid = min(T::BN, L_kv - t * T::BN);
                wave_step<D, T::NH, false, false>(st, pk_prev, vp_prev, deferred, t == t_begin, last, ks, vs,
                                                  vs_prev, fa, grp, p.scale_log2, kv_valid,
                                                  MassRange{0, 0, 0, 0, 0});
              });
  if (!wave_active) return;

#pragma unroll
  for (int j = 0; j < T::NH; ++j) {
    const int rho = qt * T::BM + (wave * T::NH + j) * 32 + l32;
    if (rho >= GL) continue;
    const int hq = g * p.G + rho / p.Ld;
    const int rr = rho % p.Ld;
    const float ltot = st[j].l + __shfl_xor(st[j].l, 32);
    float inv = 1.0f / ltot;
    float lse2 = st[j].m + __log2f(ltot);
    if (kCheckIndices && bad_index) inv = lse2 = __uint_as_float(kNanWord);
    if (p.S == 1) {
      const size_t orow = (((size_t)b * p.Ld + rr) * p.Hq + hq) * D;
      if (p.out_f32) store_row_f32<D>(reinterpret_cast<float*>(p.o_dec) + orow, st[j], inv, grp);
      else store_row_bf16<D>(reinterpret_cast<uint16_t*>(p.o_dec) + orow, st[j], inv, grp);
      if (p.lse_dec && grp == 0) p.lse_dec[((size_t)b * p.Hq + hq) * p.Ld + rr] = lse2 * kLn2;
    } else {
      const size_t row = (((size_t)sp * p.B + b) * p.Hq + hq) * p.Ld + rr;
      store_row_f32<D>(p.o_part + row * D, st[j], inv, grp);
      if (grp == 0) p.lse_part[row] = lse2;
    }
  }
}

// ---------------------------------------------------------------------------
// Eq. 5, first sum, one workgroup per (b, n, h): the query rows of head h and
// their final LSE are staged in LDS (up to 128 rows per pass), and the 4 waves
// split the C content keys in 32-key blocks, so every key row is read from HBM
// once.  S = Q_q K_c^T on MFMA (A: query rows from LDS, B: key rows from
// global memory, the next block's prefetched), each key's mass exp2(S*scale -
// lse2(row)) summed in the lane that holds the key.  The head's sum is added
// in place to its per-head second sum (written by the prefill), or replaces
// it for the query-to-chunk score; head_sum_rank_kernel then sums the heads.
// Query row r's 16-byte chunk c sits at chunk c ^ (r % CH) of its LDS row, so
// that the 16 lanes of a ds_read_b128 pass (16 rows, one chunk) hit 16
// different bank groups.
template <int D>
__global__ __launch_bounds__(256) void escore2_bf16_kernel(EscoreArgs p) {
  constexpr int KS = D / 16, CH = D / 8, QB = 128;
  __shared__ __attribute__((aligned(16))) uint16_t qs[QB * D];
  __shared__ __attribute__((aligned(16))) float ls[QB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, grp = lane >> 5;
  const size_t bnh = blockIdx.x;   // (b * N + n) * Hq + h
  const int h = (int)(bnh % p.Hq);
  const size_t bn = bnh / p.Hq;
  const int b = (int)(bn / p.N);
  const int g = h / p.G, C1 = p.C + 1;
  const size_t qm_base = (p.qm_per_chunk ? bn : (size_t)b) * (size_t)(p.Lq + p.Lm);
  const uint16_t* kbase = p.k_cache + ((bn * p.Hkv + g) * C1 + 1) * D;   // content row j at kbase + j*D
  const float* lse = p.lse_q + bnh * p.Lq;
  float* ph = p.part_io + bnh * p.C;
  const int nkb = (p.C + 31) / 32;
  auto load_k = [&](int kb, bf16x8 (&kf)[KS]) {
    const int j = kb * 32 + l32;
    const uint16_t* src = j < p.C ? kbase + (size_t)j * D : nullptr;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[ks] = src ? __builtin_bit_cast(bf16x8, ld16(src + 16 * ks + 8 * grp)) : bf16x8{0};
  };
  for (int r0 = 0; r0 < p.Lq; r0 += QB) {
    const int nr = min(QB, p.Lq - r0);
    if (r0 > 0) __syncthreads();   // the previous pass is done with qs, ls
    for (int u = tid; u < QB * CH; u += 256) {
      const int r = u / CH, c = u % CH;
      const u32x4 v = r < nr ? ld16(p.q_qm + ((qm_base + r0 + r) * p.Hq + h) * D + 8 * c) : u32x4{0u, 0u, 0u, 0u};
      st16(qs + r * D + 8 * (c ^ (r % CH)), v);
    }
    for (int r = tid; r < QB; r += 256) ls[r] = r < nr ? lse[r0 + r] : INFINITY;
    __syncthreads();
    bf16x8 kf[KS], kn[KS];
    if (wave < nkb) load_k(wave, kf);
    for (int kb = wave; kb < nkb; kb += 4) {
      if (kb + 4 < nkb) load_k(kb + 4, kn);
      float colsum = 0.f;
#pragma unroll
      for (int qb = 0; qb < QB / 32; ++qb) {
        if (qb * 32 >= nr) break;
        const int row = qb * 32 + l32;
        f32x16 sacc = f32x16{0};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 qa = __builtin_bit_cast(bf16x8, ld16(qs + row * D + 8 * ((2 * ks + grp) ^ (row % CH))));
          sacc = mfma32x32x16(qa, kf[ks], sacc);
        }
        // Row (query) of element r: qb*32 + 8*(r/4) + 4*grp + r%4.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(ls + qb * 32 + 8 * i + 4 * grp);
#pragma unroll
          for (int e = 0; e < 4; ++e) colsum += fast_exp2(sacc[4 * i + e] * p.scale_log2 - l4[e]);
        }
      }
      const float v = colsum + __shfl_xor(colsum, 32);
      const int j = kb * 32 + l32;
      if (grp == 0 && j < p.C) ph[j] = (p.q2c && r0 == 0) ? v : ph[j] + v;
      if (kb + 4 < nkb) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kf[ks] = kn[ks];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers.
template <int D>
static hipError_t launch_prefill_d(const PrefillArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(prefill_bf16_kernel<D>, dim3(a.total), dim3(Tile<D>::NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_prefill_bf16(const PrefillArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? launch_prefill_d<128>(a, s) : launch_prefill_d<64>(a, s);
}

template <int D>
static hipError_t launch_decode_d(const DecodeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(decode_bf16_kernel<D>, dim3(a.total), dim3(Tile<D>::NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_decode_bf16(const DecodeArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? launch_decode_d<128>(a, s) : launch_decode_d<64>(a, s);
}

template <int D>
static hipError_t launch_escore_d(const EscoreArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(escore2_bf16_kernel<D>, dim3(a.B * a.N * a.Hq), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_escore_bf16(const EscoreArgs& a, int head_dim, hipStream_t s) {
  return head_dim == 128 ? launch_escore_d<128>(a, s) : launch_escore_d<64>(a, s);
}

}  // namespace pd
