// Chunk staging: the raw rows of one 64-token chunk are fetched from HBM once
// per workgroup into registers (16 bytes per load, coalesced), one chunk
// ahead of the computation, then written to LDS where every wave reads the
// operand fragments it needs.  This hides the global-memory latency behind a
// whole chunk of work and removes the redundant per-wave reads.
#pragma once
#include "flex_common.hpp"

namespace flex {

// Row-major staging of a [64 x COLS] io-typed block with a padded row.
template <class IO, int COLS, int NT, int ROWS = CHUNK>
struct RowStage {
  static constexpr int VEC = 16 / sizeof(IO);           // elements per 16-byte vector
  static constexpr int VPR = COLS / VEC;                 // vectors per row
  static constexpr int NV = ROWS * VPR;                  // vectors per chunk
  static constexpr int PER = (NV + NT - 1) / NT;         // vectors per thread
  static constexpr int LD = COLS + VEC;                  // LDS row stride (elements), keeps 16 B alignment
  static constexpr int LDS_ELEMS = ROWS * LD;
  uint4 r[PER];
  uint32_t okm;   // bit i: vector i belongs to this thread and to a row below n

  // rows: this (b,h) slice's [N, COLS] rows; rows at or beyond n read as zero.
  // The loads are unconditional, from a clamped in-range row, so that nothing
  // writes their destination registers while they are in flight (a zeroing
  // branch would make the compiler wait for each load right away); the
  // out-of-range vectors are zeroed when they are stored.  n >= 1.
  __device__ __forceinline__ void fetch(const IO* __restrict__ rows, int tok0, int n) {
    okm = 0u;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v0 = threadIdx.x + i * NT;
      const int v = v0 < NV ? v0 : NV - 1;
      const int t = v / VPR, c = v % VPR;
      const int row = tok0 + t < n ? tok0 + t : n - 1;
      r[i] = *reinterpret_cast<const uint4*>(rows + (size_t)row * COLS + c * VEC);
      if (v0 < NV && tok0 + t < n) okm |= 1u << i;
    }
  }
  __device__ __forceinline__ uint4 vec(int i) const {
    return ((okm >> i) & 1u) ? r[i] : make_uint4(0u, 0u, 0u, 0u);
  }
  // keeps the fetched rows' loads without storing them anywhere (loads whose
  // only purpose is to bring the rows into the caches for a later kernel)
  __device__ __forceinline__ void touch() const {
#pragma unroll
    for (int i = 0; i < PER; ++i) asm volatile("" ::"v"(r[i].x), "v"(r[i].y), "v"(r[i].z), "v"(r[i].w));
  }
  __device__ __forceinline__ void store(IO* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v = threadIdx.x + i * NT;
      if (v < NV) {
        const int t = v / VPR, c = v % VPR;
        *reinterpret_cast<uint4*>(lds + t * LD + c * VEC) = vec(i);
      }
    }
  }
  // Squared norms are summed in fp32 for bf16 rows and in float64 for fp32
  // rows (the fp32 path's norm factor is formed in float64).
  typedef typename SsqType<IO>::type Ssq;
  // store, plus the squared norm of every row into ssq[ROWS] (the VPR vectors
  // of a row sit in VPR consecutive lanes: summed with lane shuffles)
  __device__ __forceinline__ void store(IO* lds, Ssq* ssq) const {
    store(lds, ssq, [](int, Ssq s) { return s; });
  }
  // store, plus f(row, squared norm of the row) into out[ROWS]
  template <class OUT, class F>
  __device__ __forceinline__ void store(IO* lds, OUT* out, F f) const {
    store_idx(lds, out, [&](int, int t, Ssq s) { return f(t, s); });
  }
  // as store, with f also given the index i < PER of the thread's vector
  template <class OUT, class F>
  __device__ __forceinline__ void store_idx(IO* lds, OUT* out, F f) const {
    static_assert(NT % VPR == 0 && VPR <= WAVE, "a row's vectors must share a wave");
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v = threadIdx.x + i * NT;
      Ssq s = 0;
      if (v < NV) {
        const int t = v / VPR, c = v % VPR;
        const uint4 x = vec(i);
        *reinterpret_cast<uint4*>(lds + t * LD + c * VEC) = x;
        const IO* e = reinterpret_cast<const IO*>(&x);
#pragma unroll
        for (int j = 0; j < VEC; ++j) { const Ssq y = io_to_float(e[j]); s += y * y; }
      }
      if constexpr (sizeof(Ssq) == 4) {
        s = lane_sum<VPR>(s);
      } else {
#pragma unroll
        for (int o = 1; o < VPR; o <<= 1) s += __shfl_xor(s, o);
      }
      if (v < NV && v % VPR == 0) out[v / VPR] = f(i, v / VPR, s);
    }
  }
  // transposed store: ldsT[col][token] with row stride LDT (operand type T)
  template <class T, int LDT>
  __device__ __forceinline__ void store_t(T* ldsT) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int v = threadIdx.x + i * NT;
      if (v < NV) {
        const int t = v / VPR, c = v % VPR;
        const uint4 x = vec(i);
        const IO* e = reinterpret_cast<const IO*>(&x);
#pragma unroll
        for (int j = 0; j < VEC; ++j) ldsT[(c * VEC + j) * LDT + t] = io_to_op<T>(e[j]);
      }
    }
  }
};

// Operand fragment of 8 consecutive columns [c0, c0+8) of LDS row `row`.
__device__ __forceinline__ void lds_row8(Frag<__bf16>& f, const u16* row, int c0) {
  f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(row + c0));
}
__device__ __forceinline__ void lds_row8(Frag<float>& f, const float* row, int c0) {
  const float4 a = *reinterpret_cast<const float4*>(row + c0);
  const float4 b = *reinterpret_cast<const float4*>(row + c0 + 4);
  f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
  f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
}

// fp32 path: one projection tile on the FP64 matrix cores (operand layouts in
// FreqSlice<float>).  ROWS_AS_TOKENS = false: the tile holds frequencies 4g+i
// (rows) x token r (cols), as the bf16 tile of project_tile_lds; true: tokens
// 4g+i x frequency r, as project_rows_lds (the X rows are then permuted so
// that accumulator slot i of lane group g is token 4g + i).
template <int D, int FW, bool NS, int LD, bool ROWS_AS_TOKENS>
__device__ __forceinline__ void project_f64(const FreqSlice<float, D, FW, NS>& fs, const float* X, int tt,
                                            f64x4 (&p)[FreqSlice<float, D, FW, NS>::PR]) {
  typedef FreqSlice<float, D, FW, NS> FS;
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const float* xr = X + (tt * 16 + (ROWS_AS_TOKENS ? f64_tile_row(r) : r)) * LD;
#pragma unroll
  for (int pr = 0; pr < FS::PR; ++pr) p[pr] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int ks = 0; ks < FS::KS; ++ks) {
    const double x = xr[4 * ks + g];
#pragma unroll
    for (int pr = 0; pr < FS::PR; ++pr)
      p[pr] = ROWS_AS_TOKENS ? __builtin_amdgcn_mfma_f64_16x16x4f64(x, fs.wr[pr][ks], p[pr], 0, 0, 0)
                             : __builtin_amdgcn_mfma_f64_16x16x4f64(fs.wt[pr][ks], x, p[pr], 0, 0, 0);
  }
}

// Projection of one 16-token tile (rows staged in LDS, row stride LD) onto a
// wave's frequency slice, plus the squared row norm (summed over lane groups).
template <class T, int D, int FW, bool NS, int LD, class S>
__device__ __forceinline__ void project_tile_lds(const FreqSlice<T, D, FW, NS>& fs,
                                                 const typename Io<T>::type* X, const S* ssq_rows,
                                                 int tt, ProjT<T> (&p)[FreqSlice<T, D, FW, NS>::PR],
                                                 S& ssq) {
  typedef FreqSlice<T, D, FW, NS> FS;
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  if constexpr (!IsBf16<T>::value) {
    project_f64<D, FW, NS, LD, false>(fs, X, tt, p);
  } else {
    const typename Io<T>::type* row = X + (tt * 16 + r) * LD;
#pragma unroll
    for (int pr = 0; pr < FS::PR; ++pr) p[pr] = zero4();
#pragma unroll
    for (int ks = 0; ks < FS::KD; ++ks) {
      Frag<T> x;
      lds_row8(x, row, ks * 32 + 8 * g);
#pragma unroll
      for (int pr = 0; pr < FS::PR; ++pr)
#pragma unroll
        for (int sp = 0; sp < FS::NSPLIT; ++sp) mma(p[pr], fs.w[sp][pr][ks], x);
    }
  }
  ssq = ssq_rows[tt * 16 + r];
}

template <class T, int D, int FW, int NW, bool NS, int CH_ = CHUNK>
struct Shape {
  static constexpr int CH = CH_;            // tokens per chunk
  static constexpr int TT = CH / 16;        // token tiles per chunk
  static constexpr int M = FW * NW;
  static constexpr int FT = FW / 16;        // frequency tiles per wave
  static constexpr int FC = 2 * FT;         // feature tiles per wave
  static constexpr int DV = D;
  static constexpr int DVT = DV / 16;       // value tiles
  static constexpr int DVT1 = DVT + 1;      // + the normaliser tile
  static constexpr int KT = CH / 32;        // k-steps over the tokens of a chunk
  static constexpr int PR = NS ? 2 * FT : FT;
  static constexpr int NT = NW * WAVE;      // threads per workgroup
  // fp32 floats of one wave's state, one (b,h,segment) block of the workspace
  static constexpr int WAVE_STATE = FC * DVT1 * WAVE * 4;
  static constexpr int STATE = NW * WAVE_STATE;
  // LDS row strides (elements); multiples of 4 keep 8/16-byte alignment
  static constexpr int TPAD = CH + 4;
  static constexpr int RPAD = DVT1 * 16 + 4;
};

// Fragment with 1 in row/column 0 and 0 elsewhere: as the value operand it
// appends the ones column of [V | 1] that produces the normaliser.
template <class T>
__device__ __forceinline__ Frag<T> ones_col0() {
  Frag<T> f;
  const float v = (threadIdx.x % 16) == 0 ? 1.0f : 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.set(j, v);
  return f;
}

// Operand fragment over the chunk's tokens from a token-contiguous LDS row:
// slots j<4 take tokens 32ks+4g+j, slots j>=4 tokens 32ks+16+4g+j-4.  This is
// the token order of a pair of accumulator tiles (see pair_tiles).
template <class T>
__device__ __forceinline__ Frag<T> lds_tok_frag(const T* row, int ks) {
  const int g = (threadIdx.x % WAVE) / 16;
  Frag<T> f;
  const T* a = row + 32 * ks + 4 * g;
  const T* b = a + 16;
#pragma unroll
  for (int j = 0; j < 4; ++j) { f.set(j, (float)a[j]); f.set(4 + j, (float)b[j]); }
  return f;
}
template <>
__device__ __forceinline__ Frag<__bf16> lds_tok_frag<__bf16>(const __bf16* row, int ks) {
  const int g = (threadIdx.x % WAVE) / 16;
  const __bf16* a = row + 32 * ks + 4 * g;
  bf16x4 lo = *reinterpret_cast<const bf16x4*>(a);
  bf16x4 hi = *reinterpret_cast<const bf16x4*>(a + 16);
  Frag<__bf16> f;
  f.v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return f;
}

// Two accumulator tiles whose rows are consecutive 16-blocks of a contraction
// index, as one operand fragment (slots 0..3 from the first, 4..7 from the second).
template <class T>
__device__ __forceinline__ Frag<T> pair_tiles(const f32x4& a, const f32x4& b) {
  Frag<T> f;
#pragma unroll
  for (int i = 0; i < 4; ++i) { f.set(i, a[i]); f.set(4 + i, b[i]); }
  return f;
}

// Projection of one 16-token tile with the tokens as rows: p[pr] holds rows =
// tokens tt*16 + 4g + i and cols = frequency (lane % 16) of projection tile
// pr.  The operands of project_tile_lds are swapped (the register layouts of
// the two MFMA operands are the same), so the frequency fragments are shared.
template <class T, int D, int FW, bool NS, int LD>
__device__ __forceinline__ void project_rows_lds(const FreqSlice<T, D, FW, NS>& fs,
                                                 const typename Io<T>::type* X, int tt,
                                                 ProjT<T> (&p)[FreqSlice<T, D, FW, NS>::PR]) {
  typedef FreqSlice<T, D, FW, NS> FS;
  if constexpr (!IsBf16<T>::value) {
    project_f64<D, FW, NS, LD, true>(fs, X, tt, p);
  } else {
    const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
    const typename Io<T>::type* row = X + (tt * 16 + r) * LD;
#pragma unroll
    for (int pr = 0; pr < FS::PR; ++pr) p[pr] = zero4();
#pragma unroll
    for (int ks = 0; ks < FS::KD; ++ks) {
      Frag<T> x;
      lds_row8(x, row, ks * 32 + 8 * g);
#pragma unroll
      for (int pr = 0; pr < FS::PR; ++pr)
#pragma unroll
        for (int sp = 0; sp < FS::NSPLIT; ++sp) mma(p[pr], x, fs.w[sp][pr][ks]);
    }
  }
}

// Features of a wave's frequency slice for the 32 tokens of k-step ks, with
// the tokens as the contraction index: out[2ft] (cos-type) and out[2ft+1]
// (sin-type) have cols = the feature (lane % 16) and k = tokens in the order
// of pair_tiles / lds_tok_frag.  sc[t] is the per-token scale (0 for tokens
// past the end).  Used where a feature map only enters contractions over
// tokens (state sums), which then need no transpose through LDS.  fv: as in
// features (slice frequencies ft*16 + lane%16 >= fv give zero features).
template <class T, int D, int FW, bool NS, int LD>
__device__ __forceinline__ void feature_frags_rows(const FreqSlice<T, D, FW, NS>& fs,
                                                   const typename Io<T>::type* X, const float* sc,
                                                   int ks, Frag<T> (&out)[2 * (FW / 16)], int fv = FW) {
  typedef FreqSlice<T, D, FW, NS> FS;
  constexpr int FT = FW / 16;
  const int g = (threadIdx.x % WAVE) / 16;
  f32x4 fc[2][FT], fsn[2][FT];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int tt = 2 * ks + hh;
    ProjT<T> p[FS::PR];
    project_rows_lds<T, D, FW, NS, LD>(fs, X, tt, p);
    const float4 s4 = *reinterpret_cast<const float4*>(sc + tt * 16 + 4 * g);
    const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
    for (int ft = 0; ft < FT; ++ft)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float s1, c1;
        sincos_rev(p[ft][i], s1, c1);
        const float m = NS ? sv[i] * cos_rev(p[FT + ft][i]) : sv[i];
        fc[hh][ft][i] = c1 * m;
        fsn[hh][ft][i] = s1 * m;
      }
  }
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) {
    out[2 * ft] = pair_tiles<T>(fc[0][ft], fc[1][ft]);
    out[2 * ft + 1] = pair_tiles<T>(fsn[0][ft], fsn[1][ft]);
  }
  if (fv < FW) {   // this lane's frequency is slice frequency ft*16 + lane % 16
#pragma unroll
    for (int ft = 0; ft < FT; ++ft)
      if (ft * 16 + (int)(threadIdx.x % 16) >= fv) { out[2 * ft].zero(); out[2 * ft + 1].zero(); }
  }
}

// ---------------------------------------------------------------------------
// Transposes through LDS with the gfx950 transpose load.  An accumulator tile
// holds column n = lane % 16 and rows m = 4g + i (g = lane / 16); written as
// bf16 into an [n][m]-major block it is one 8-byte store per lane.  Reading
// that block back with ds_read_b64_tr_b16 gives an operand whose lane is m and
// whose k index is n: within each group of 16 lanes, slot j of lane i receives
// element i % 4 of the 4-element row addressed by lane 4j + i / 4, so lane
// (g, i) addresses row kb + i / 4, columns m0 + 4 (i % 4) .. + 3, and receives
// column m0 + i of rows kb .. kb + 3.  The fp32 operand type keeps plain
// element-wise accesses of the same layouts.
// ---------------------------------------------------------------------------
typedef short tr_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) tr_v4i16 lds_tr_v4i16;

// Rows 4g..4g+3 of an accumulator tile (values v) into L[n][m0 + 4g + i],
// n = n0 + lane % 16.
template <class T>
__device__ __forceinline__ void store_tile_nm(T* L, int ld, int n0, int m0, const f32x4& v) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  T* o = L + (n0 + r) * ld + m0 + 4 * g;
  if constexpr (IsBf16<T>::value) {
    const bf16x4 b = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
    *reinterpret_cast<bf16x4*>(o) = b;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = v[i];
  }
}

// The two halves of an operand fragment (slots 0..3 and 4..7, each four rows
// 4g..4g+3 of one tile) into L[n][m0a + 4g + i] and L[n][m0b + 4g + i].
template <class T>
__device__ __forceinline__ void store_frag_nm(T* L, int ld, int n0, int m0a, int m0b, const Frag<T>& f) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  T* row = L + (n0 + r) * ld + 4 * g;
  if constexpr (IsBf16<T>::value) {
    const uint4 w = __builtin_bit_cast(uint4, f.v);
    *reinterpret_cast<uint2*>(row + m0a) = make_uint2(w.x, w.y);
    *reinterpret_cast<uint2*>(row + m0b) = make_uint2(w.z, w.w);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) { row[m0a + i] = f.raw(i); row[m0b + i] = f.raw(4 + i); }
  }
}

// Operand fragment stored by store_frag_nm, read back in the same layout:
// lane row n0 + lane % 16, slots 0..3 from columns m0a + 4g .. + 3, slots
// 4..7 from m0b + 4g .. + 3.
template <class T>
__device__ __forceinline__ Frag<T> load_frag_nm(const T* L, int ld, int n0, int m0a, int m0b) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const T* row = L + (n0 + r) * ld + 4 * g;
  Frag<T> f;
  if constexpr (IsBf16<T>::value) {
    const uint2 a = *reinterpret_cast<const uint2*>(row + m0a);
    const uint2 b = *reinterpret_cast<const uint2*>(row + m0b);
    f.v = __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) { f.set(i, row[m0a + i]); f.set(4 + i, row[m0b + i]); }
  }
  return f;
}

// Operand fragment with lane m = m0 + lane % 16 and k slots 0..3 = rows
// kb0 .. kb0+3, slots 4..7 = rows kb1 .. kb1+3 of an [k][m]-major block
// (kb0, kb1 may differ between lane groups).
template <class T>
__device__ __forceinline__ Frag<T> lds_tr_frag(const T* L, int ld, int kb0, int kb1, int m0) {
  const int i = (threadIdx.x % WAVE) % 16;
  Frag<T> f;
  if constexpr (IsBf16<T>::value) {
    const int off = (i / 4) * ld + m0 + 4 * (i % 4);
    const tr_v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(L + kb0 * ld + off));
    const tr_v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_tr_v4i16*)(L + kb1 * ld + off));
    f.v = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f.set(j, L[(kb0 + j) * ld + m0 + i]);
      f.set(4 + j, L[(kb1 + j) * ld + m0 + i]);
    }
  }
  return f;
}

}  // namespace flex
