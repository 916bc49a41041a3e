// Device helpers shared by the backward kernels (flex_bwd.hip, flex_bwd_dq.hip):
// feature fragments with their P2-derivative, the normaliser rows of the
// backward states, per-token scalars, state tile layouts, the feature-map
// chain rule and the frequency-gradient partials.
#pragma once
#include "flex_common.hpp"
#include "flex_kernels.hpp"
#include "flex_stage.hpp"

namespace flex {

// Feature fragment (as in the forward) plus, for the nonstationary variant,
// the fragment of d phi / d P2 up to sign: slots [s e sin P2 cos P1 | s e sin P2 sin P1].
// fv: as in features (slice frequencies >= fv give zero fragments).
template <class T, int FT, bool NS, class P>
__device__ __forceinline__ void features_psi(const P (&p)[NS ? 2 * FT : FT], int ft, float scale,
                                             Frag<T>& phi, Frag<T>& psi, int fv = FT * 16) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float s1, c1;
    sincos_rev(p[ft][i], s1, c1);
    if (NS) {
      float s2, c2;
      sincos_rev(p[FT + ft][i], s2, c2);
      const float sc = scale * c2, ss = scale * s2;
      phi.set(i, c1 * sc);
      phi.set(4 + i, s1 * sc);
      psi.set(i, c1 * ss);
      psi.set(4 + i, s1 * ss);
    } else {
      phi.set(i, c1 * scale);
      phi.set(4 + i, s1 * scale);
    }
  }
  if (fv < FT * 16) {
    mask_features(phi, ft, fv);
    if (NS) mask_features(psi, ft, fv);
  }
}

// -x as a two-term operand split (hi, lo): exact to about 16 bits on the bf16
// path.  The backward states carry the normaliser products in two rows of the
// normaliser tile (value columns dv and dv+1) so that delta_i is not rounded
// to bf16 on its way into them.
template <class T>
__device__ __forceinline__ void neg_split(float x, float& hi, float& lo) {
  if (IsBf16<T>::value) {
    hi = (float)(__bf16)(-x);
    lo = -x - hi;
  } else {
    hi = -x;
    lo = 0.f;
  }
}
template <class T>
__device__ __forceinline__ Frag<T> ones_col01() {
  Frag<T> f;
  const float v = (threadIdx.x % 16) < 2 ? 1.0f : 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) f.set(j, v);
  return f;
}
// Normaliser-row operand over chunk tokens k-step ks: rows dv, dv+1 hold the
// split of -delta_t for the tokens of the paired-tile order.
template <class T>
__device__ __forceinline__ Frag<T> delta_rows(const float (*GS)[2], int ks) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  Frag<T> f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int t = 32 * ks + (j >= 4 ? 16 : 0) + 4 * g + (j & 3);
    float hi, lo;
    neg_split<T>(GS[t][1], hi, lo);
    f.set(j, r == 0 ? hi : (r == 1 ? lo : 0.f));
  }
  return f;
}

// Per-token (1/den, delta) of token tok0 + (thread mod ch), loaded from a
// clamped in-range index so that the load is unconditional (ok: the thread
// holds a token of the chunk below n; others are zeroed where they are stored).
__device__ __forceinline__ float2 load_gs(const float* gst, int tok0, int n, int ch, bool& ok) {
  const int t = tok0 + (int)(threadIdx.x % ch);
  ok = (int)threadIdx.x < ch && t < n;
  return *reinterpret_cast<const float2*>(gst + (size_t)min(t, n - 1) * 2);
}

// Register-dump layout of the [dv' x features] states: tile (dt, global feature
// tile w*FC + fc), lane, 4 floats.  It does not depend on how the waves split
// the frequencies, so kernels with different splits share the states.
template <class SH>
__device__ __forceinline__ size_t state_off(int w, int dt, int fc, int l) {
  constexpr int NFT = SH::M / 8;   // feature tiles of the whole [cos | sin] feature vector
  return ((size_t)(dt * NFT + w * SH::FC + fc) * WAVE + l) * 4;
}

// Tile (dt, fc) of this wave's [dv' x features] key-side state read from a
// forward segment-state block.  The forward keeps [features x dv'] tiles
// (feature tile F, value tile dt; rows = features, cols = value columns) in
// register-dump order, with the normaliser in value column dv; the backward
// tile is its transpose, with the normaliser in both rows dv and dv+1 (the
// two rows that take the split of -delta).
template <class SH>
__device__ __forceinline__ f32x4 fwd_state_tile_t(const float* blk, int w, int dt, int fc) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const float* tile = blk + (size_t)((w * SH::FC + fc) * SH::DVT1 + dt) * WAVE * 4;
  f32x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int vl = 4 * g + i;                     // value column within tile dt
    const bool norm = dt == SH::DVT;
    const int col = norm ? 0 : vl;                // forward column of this value
    // forward element (feature r, column col): lane col + 16 (r / 4), slot r % 4
    const float x = tile[(col + 16 * (r / 4)) * 4 + (r % 4)];
    v[i] = (!norm || vl < 2) ? x : 0.f;
  }
  return v;
}

// Chain rule through one wave's features for frequency tile ft, token tile tt:
// dP (per radian) for the projection rows, and <phi, dphi> summed over this
// lane's slots.
template <class T, int FT, bool NS>
__device__ __forceinline__ float feature_grad(const Frag<T>& phi, const Frag<T>& psi,
                                              const f32x4& da, const f32x4& db, f32x4& dp1, f32x4& dp2) {
  float gsum = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = phi.get(i), b = phi.get(4 + i);
    dp1[i] = a * db[i] - b * da[i];
    if (NS) dp2[i] = -(psi.get(i) * da[i] + psi.get(4 + i) * db[i]);
    gsum += a * da[i] + b * db[i];
  }
  return gsum;
}

// The per-wave frequency-gradient partial dW'[rows][d] lives in LDS in
// register-dump order (tile, lane, 4 floats).  Each chunk's product for
// projection-row tile pr is formed with the LDS tiles as the MFMA's
// accumulator input (one 16-byte read and write per lane and tile), so the
// sum takes no vector ALU work.
template <int D, class T>
__device__ __forceinline__ void dw_mma_row(float* dwl, int pr, const Frag<T>& dpt, const Frag<T> (&x)[D / 16]) {
  const int l = threadIdx.x % WAVE;
  f32x4 c[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) c[dt] = *reinterpret_cast<const f32x4*>(dwl + ((pr * (D / 16) + dt) * WAVE + l) * 4);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) mma(c[dt], dpt, x[dt]);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) *reinterpret_cast<f32x4*>(dwl + ((pr * (D / 16) + dt) * WAVE + l) * 4) = c[dt];
}

// Write a wave's frequency-gradient partial tiles DW[pr][dt] (rows = projection
// rows, cols = d) into the canonical layout [matrix][m][d].
template <class SH, int D, int FW, bool NS>
__device__ __forceinline__ void dump_dw(float* out, const float* dwl, int f0) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
#pragma unroll
  for (int pr = 0; pr < SH::PR; ++pr)
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(dwl + ((pr * (D / 16) + dt) * WAVE + l) * 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int mat = pr >= SH::FT ? 1 : 0;
        const int f = f0 + (pr % SH::FT) * 16 + 4 * g + i;
        out[((size_t)mat * SH::M + f) * D + dt * 16 + r] = v[i];
      }
    }
}

// The query side's partial is handed to the dK/dV sweep in tile-major order
// [matrix][frequency tile][d tile][lane][4], which does not depend on how a
// kernel's waves split the frequencies: the dK/dV sweep starts its own
// partial from it, so one partial per workgroup position holds both sides.
template <class SH, int D>
__device__ __forceinline__ size_t dw_tile_off(int w, int pr, int dt, int l) {
  constexpr int NFT = SH::M / 16;   // frequency tiles of one matrix
  const int mat = pr / SH::FT, ft = pr % SH::FT;
  return ((((size_t)mat * NFT + w * SH::FT + ft) * (D / 16) + dt) * WAVE + l) * 4;
}

}  // namespace flex
