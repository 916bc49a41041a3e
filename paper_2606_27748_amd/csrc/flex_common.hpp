// Device building blocks shared by the gfx950 kernels of the RFF linear
// attention library: MFMA fragments, frequency loading, the projection onto
// the frequencies and the fused trigonometric feature epilogue.
//
// Orientation used throughout ("token-column"): the projection is computed as
// P^T = W X^T with v_mfma_f32_16x16x32_bf16 (or eight v_mfma_f32_16x16x4f32 on
// the fp32 path), so a 16x16 accumulator tile holds 16 frequencies x 16 tokens
// and lane l owns token l%16 and frequencies 4*(l/16)+i, i=0..3.  The feature
// epilogue turns one such tile into one 8-wide MFMA operand fragment per lane:
// slots j=0..3 hold the cos (stationary) or cos P1 cos P2 (nonstationary)
// features of frequencies 4g+j and slots j=4..7 the matching sin /
// sin P1 cos P2 features (g = l/16).  Both operands of every contraction over
// features use this same slot -> feature map, so no shuffle is needed.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flex {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

constexpr int WAVE = 64;
constexpr int CHUNK = 64;          // tokens per chunk
constexpr int TT = CHUNK / 16;     // token tiles per chunk
constexpr float INV_2PI = 0.15915494309189535f;

// Workgroup -> (segment, b*H+h) for a 1-D grid of nseg * BH workgroups.
// Consecutive workgroup ids are dealt round-robin to the 8 XCDs, each with its
// own L2; the mapping gives every XCD a contiguous range of the list ordered
// by (head, batch, segment), so the per-head frequency fragments that every
// chunk reloads are shared by the workgroups of few heads in each L2.
constexpr int NUM_XCD = 8;
struct WgCoord {
  int seg, bh;
};
__device__ __forceinline__ WgCoord wg_coord(int nseg, int H, int BH) {
  const int T = nseg * BH;
  const int L = blockIdx.x;
  const int idx = (T % NUM_XCD == 0) ? (L % NUM_XCD) * (T / NUM_XCD) + L / NUM_XCD : L;
  const int seg = idx % nseg, t = idx / nseg;
  const int B = BH / H;
  return {seg, (t % B) * H + t / B};
}

// ---------------------------------------------------------------------------
// Fragments: 8 operand values per lane.  Lane l supplies row/col l%16 and the
// contraction indices k(g, j) for g = l/16, j = 0..7.
// ---------------------------------------------------------------------------
template <class T> struct Frag;
template <> struct Frag<__bf16> {
  bf16x8 v;
  __device__ void zero() { for (int j = 0; j < 8; ++j) v[j] = (__bf16)0.0f; }
  __device__ void set(int j, float x) { v[j] = (__bf16)x; }
  __device__ float get(int j) const { return (float)v[j]; }
  __device__ __bf16 raw(int j) const { return v[j]; }   // stored value, no conversion
};
template <> struct Frag<float> {
  float v[8];
  __device__ void zero() { for (int j = 0; j < 8; ++j) v[j] = 0.0f; }
  __device__ void set(int j, float x) { v[j] = x; }
  __device__ float get(int j) const { return v[j]; }
  __device__ float raw(int j) const { return v[j]; }
};

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

__device__ __forceinline__ void mma(f32x4& c, const Frag<__bf16>& a, const Frag<__bf16>& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
}
// One 32-long k-step as eight k=4 MFMAs chained into a fresh accumulator,
// then one add into c.  Chaining straight into c would round a long-lived
// accumulator (a carried state) once per 4 tokens instead of once per 32,
// and over a sequential sweep of a few thousand tokens that rounding grows
// to the 1e-4 scale in the gradients.
__device__ __forceinline__ void mma(f32x4& c, const Frag<float>& a, const Frag<float>& b) {
  f32x4 t = zero4();
#pragma unroll
  for (int j = 0; j < 8; ++j) t = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], t, 0, 0, 0);
  c += t;
}

template <class T> struct IsBf16 { static constexpr bool value = false; };
template <> struct IsBf16<__bf16> { static constexpr bool value = true; };

// Projection tiles and squared row norms by operand type.  The bf16 path
// projects on MFMA in fp32 (revolutions); the fp32 path forms the projection
// and the squared norms in float64, so that the phase handed to the
// trigonometric functions is exact to float64 rounding whatever its size.
template <class T> struct ProjTile { typedef f32x4 type; };
template <> struct ProjTile<float> { typedef f64x4 type; };
template <class T> using ProjT = typename ProjTile<T>::type;
template <class T> struct SsqType { typedef float type; };
template <> struct SsqType<float> { typedef double type; };

// Storage type of the io tensors for an operand type.
template <class T> struct Io;
template <> struct Io<__bf16> { typedef u16 type; };
template <> struct Io<float> { typedef float type; };

__device__ __forceinline__ float bf16_bits_to_float(u16 b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
__device__ __forceinline__ u16 float_to_bf16_bits(float x) {
  __bf16 h = (__bf16)x;
  return __builtin_bit_cast(u16, h);
}
__device__ __forceinline__ float io_to_float(u16 b) { return bf16_bits_to_float(b); }
__device__ __forceinline__ float io_to_float(float x) { return x; }
// An io element as an operand element of type T (bit copy when the types agree).
template <class T> __device__ __forceinline__ T io_to_op(u16 b);
template <> __device__ __forceinline__ __bf16 io_to_op<__bf16>(u16 b) { return __builtin_bit_cast(__bf16, b); }
template <> __device__ __forceinline__ float io_to_op<float>(u16 b) { return bf16_bits_to_float(b); }
template <class T> __device__ __forceinline__ T io_to_op(float x) { return (T)x; }
template <class S> __device__ __forceinline__ S float_to_io(float x);
template <> __device__ __forceinline__ u16 float_to_io<u16>(float x) { return float_to_bf16_bits(x); }
template <> __device__ __forceinline__ float float_to_io<float>(float x) { return x; }

// Load 8 consecutive io elements starting at p (16-byte aligned for bf16,
// 32-byte aligned for fp32) into a fragment; `ok` false gives zeros.
__device__ __forceinline__ void load8(Frag<__bf16>& f, const u16* p, bool ok) {
  if (ok) {
    uint4 r = *reinterpret_cast<const uint4*>(p);
    f.v = __builtin_bit_cast(bf16x8, r);
  } else {
    f.zero();
  }
}
__device__ __forceinline__ void load8(Frag<float>& f, const float* p, bool ok) {
  if (ok) {
    float4 a = *reinterpret_cast<const float4*>(p);
    float4 b = *reinterpret_cast<const float4*>(p + 4);
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
  } else {
    f.zero();
  }
}

// Cross-lane sums in registers (no LDS round trip).
// lane_sum<N>: sum over each aligned group of N consecutive lanes (N = 1..16),
// every lane of the group receives it.  DPP quad permutes give the pair and
// quad sums, row_half_mirror (lane i <-> 7-i within 8) the 8-lane sum once all
// lanes of a quad agree, row_mirror (i <-> 15-i) the 16-lane sum likewise.
__device__ __forceinline__ float dpp_add(float x, int ctrl_sel) {
  const int v = __builtin_bit_cast(int, x);
  int y;
  switch (ctrl_sel) {
    case 0: y = __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false); break;   // quad_perm [1,0,3,2]
    case 1: y = __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false); break;   // quad_perm [2,3,0,1]
    case 2: y = __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false); break;  // row_half_mirror
    default: y = __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false); break; // row_mirror
  }
  return x + __builtin_bit_cast(float, y);
}
template <int N>
__device__ __forceinline__ float lane_sum(float x) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16, "lane_sum: N in {1,2,4,8,16}");
  if (N >= 2) x = dpp_add(x, 0);
  if (N >= 4) x = dpp_add(x, 1);
  if (N >= 8) x = dpp_add(x, 2);
  if (N >= 16) x = dpp_add(x, 3);
  return x;
}
// Sum over the four lane groups (lanes l, l^16, l^32, l^48).  Used off the
// hot path only (the hot sweeps reduce across lane groups through LDS).
__device__ __forceinline__ float group_sum(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// ---------------------------------------------------------------------------
// Per-wave frequency slice.  A wave owns FW consecutive frequencies starting
// at f0; its projection rows are those FW rows of W (stationary) or of W'1
// followed by the same FW rows of W'2 (nonstationary), scaled by 1/(2 pi) so
// that the projection comes out in revolutions.  On the bf16 path each row is
// held as a two-term bf16 split hi + lo (about 16 significant bits).
// ---------------------------------------------------------------------------
template <class T, int D, int FW, bool NS>
struct FreqSlice {
  static constexpr int FT = FW / 16;               // frequency tiles
  static constexpr int PR = NS ? 2 * FT : FT;      // projection row tiles
  static constexpr int KD = D / 32;                // k-steps over d
  static constexpr int NSPLIT = IsBf16<T>::value ? 2 : 1;
  Frag<T> w[NSPLIT][PR][KD];

  // W1, W2: [m, d] fp32 rows of this head.  ROWS: rows f >= rows (when
  // given) are not read and load as zero frequencies.
  template <bool ROWS = false>
  __device__ void load(const float* __restrict__ W1, const float* __restrict__ W2, int f0, int rows = 0) {
    const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
#pragma unroll
    for (int pr = 0; pr < PR; ++pr) {
      const int f = f0 + (pr % FT) * 16 + r;
      const bool second = pr >= FT;
      const bool in = !ROWS || f < rows;
      const int fr = in ? f : 0;
#pragma unroll
      for (int ks = 0; ks < KD; ++ks) {
        const int c0 = ks * 32 + 8 * g;
        const float* a = W1 + (size_t)fr * D + c0;
        float x[8];
        float4 a0 = *reinterpret_cast<const float4*>(a);
        float4 a1 = *reinterpret_cast<const float4*>(a + 4);
        x[0] = a0.x; x[1] = a0.y; x[2] = a0.z; x[3] = a0.w;
        x[4] = a1.x; x[5] = a1.y; x[6] = a1.z; x[7] = a1.w;
        if (NS) {
          const float* b = W2 + (size_t)fr * D + c0;
          float4 b0 = *reinterpret_cast<const float4*>(b);
          float4 b1 = *reinterpret_cast<const float4*>(b + 4);
          float y[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
          for (int j = 0; j < 8; ++j) x[j] = second ? 0.5f * (x[j] - y[j]) : 0.5f * (x[j] + y[j]);
        }
        if (!in) {
#pragma unroll
          for (int j = 0; j < 8; ++j) x[j] = 0.0f;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float v = x[j] * INV_2PI;
          if (IsBf16<T>::value) {
            const float hi = (float)(__bf16)v;
            w[0][pr][ks].set(j, hi);
            w[NSPLIT - 1][pr][ks].set(j, v - hi);
          } else {
            w[0][pr][ks].set(j, v);
          }
        }
      }
    }
  }

  // Fragments in lane order, [fragment][lane]: one coalesced load per fragment.
  static constexpr int NFRAG = NSPLIT * PR * KD;
  __device__ __forceinline__ void store_frags(Frag<T>* out) const {
    const int l = threadIdx.x % WAVE;
#pragma unroll
    for (int sp = 0; sp < NSPLIT; ++sp)
#pragma unroll
      for (int pr = 0; pr < PR; ++pr)
#pragma unroll
        for (int ks = 0; ks < KD; ++ks) out[((sp * PR + pr) * KD + ks) * WAVE + l] = w[sp][pr][ks];
  }
  __device__ __forceinline__ void load_frags(const Frag<T>* in) {
    const int l = threadIdx.x % WAVE;
#pragma unroll
    for (int sp = 0; sp < NSPLIT; ++sp)
#pragma unroll
      for (int pr = 0; pr < PR; ++pr)
#pragma unroll
        for (int ks = 0; ks < KD; ++ks) w[sp][pr][ks] = in[((sp * PR + pr) * KD + ks) * WAVE + l];
  }
};

// fp32 path: float64 operands of the projection on the FP64 matrix cores
// (v_mfma_f64_16x16x4f64: A[m][k] and B[k][n] one element per lane, lane l
// supplying index l%16 at k = l/16; D holds rows l/16 + 4i, i = 0..3, of
// column l%16).  The frequencies W'/(2 pi) are formed in float64 from the fp32
// rows (W'1 = (w1 + w2)/2 and W'2 = (w1 - w2)/2 exactly), so the projection
// reaches float64 accuracy before the phase is reduced.  Two operand layouts:
//   wt: A operand of the frequency-row tile P^T = W' X^T; lane row rho holds
//       frequency 4 (rho % 4) + rho / 4, so that accumulator slot i of lane
//       group g is frequency 4g + i as in the bf16 tiles;
//   wr: B operand of the token-row tile P = X W'^T; lane row rho holds
//       frequency rho (the token rows are permuted on the X side instead).
// A prepared block holds wt then wr per lane, in the space NFRAG reserves.
__device__ __forceinline__ int f64_tile_row(int rho) { return 4 * (rho % 4) + rho / 4; }

template <int D, int FW, bool NS>
struct FreqSlice<float, D, FW, NS> {
  static constexpr int FT = FW / 16;
  static constexpr int PR = NS ? 2 * FT : FT;
  static constexpr int KD = D / 32;
  static constexpr int NSPLIT = 1;
  static constexpr int KS = D / 4;                 // f64 MFMA k-steps over d
  static constexpr int NFRAG = 2 * PR * KS / 4;    // Frag<float> units (32 bytes per lane)
  static_assert((2 * PR * KS) % 4 == 0, "whole fragment units");
  double wt[PR][KS];
  double wr[PR][KS];

  template <bool ROWS = false>
  __device__ void load(const float* __restrict__ W1, const float* __restrict__ W2, int f0, int rows = 0) {
    constexpr double INV_2PI_D = 0.15915494309189535;
    const int l = threadIdx.x % WAVE, rho = l % 16, g = l / 16;
#pragma unroll
    for (int pr = 0; pr < PR; ++pr) {
      const int ft = pr % FT;
      const bool second = pr >= FT;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int k = 4 * ks + g;
#pragma unroll
        for (int v = 0; v < 2; ++v) {
          const int f = f0 + ft * 16 + (v == 0 ? f64_tile_row(rho) : rho);
          const bool in = !ROWS || f < rows;
          const int fr = in ? f : 0;
          double w = W1[(size_t)fr * D + k];
          if (NS) {
            const double w2 = W2[(size_t)fr * D + k];
            w = second ? 0.5 * (w - w2) : 0.5 * (w + w2);
          }
          if (!in) w = 0.0;
          w *= INV_2PI_D;
          if (v == 0) wt[pr][ks] = w; else wr[pr][ks] = w;
        }
      }
    }
  }
  __device__ __forceinline__ void store_frags(Frag<float>* out) const {
    double* o = reinterpret_cast<double*>(out);
    const int l = threadIdx.x % WAVE;
#pragma unroll
    for (int pr = 0; pr < PR; ++pr)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        o[(pr * KS + ks) * WAVE + l] = wt[pr][ks];
        o[((PR + pr) * KS + ks) * WAVE + l] = wr[pr][ks];
      }
  }
  __device__ __forceinline__ void load_frags(const Frag<float>* in) {
    const double* o = reinterpret_cast<const double*>(in);
    const int l = threadIdx.x % WAVE;
#pragma unroll
    for (int pr = 0; pr < PR; ++pr)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        wt[pr][ks] = o[(pr * KS + ks) * WAVE + l];
        wr[pr][ks] = o[((PR + pr) * KS + ks) * WAVE + l];
      }
  }
};

// A-operand fragments of W'^T (rows = input dimension d, k = projection rows of
// this wave, paired tiles) in radians, in the operand type.  Used for
// dX = dP W'.  Projection row tile pr < FT is W'1 (or W), pr >= FT is W'2.
// One term (no hi + lo split, unlike the projection fragments): dP is itself
// rounded to the operand type in this product, and a relative rounding of W'
// of the same size only enters dX linearly, whereas the projection's phase
// error is multiplied by |P| inside the trigonometric functions.
template <class T, int D, int FW, bool NS>
struct WTSlice {
  static constexpr int FT = FW / 16;
  static constexpr int PR = NS ? 2 * FT : FT;
  static constexpr int KP = (PR + 1) / 2;      // k-steps over the projection rows
  static constexpr int DT = D / 16;
  static constexpr int NSPLIT = 1;
  Frag<T> w[NSPLIT][DT][KP];

  __device__ void load(const float* __restrict__ W1, const float* __restrict__ W2, int f0) {
    const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int dcol = dt * 16 + r;
#pragma unroll
      for (int ks = 0; ks < KP; ++ks) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int pr = 2 * ks + (j >= 4 ? 1 : 0);
          float v = 0.f;
          if (pr < PR) {
            const int f = f0 + (pr % FT) * 16 + 4 * g + (j & 3);
            const float x = W1[(size_t)f * D + dcol];
            if (NS) {
              const float y = W2[(size_t)f * D + dcol];
              v = pr >= FT ? 0.5f * (x - y) : 0.5f * (x + y);
            } else {
              v = x;
            }
          }
          w[0][dt][ks].set(j, v);   // rounded to the operand type (RNE)
        }
      }
    }
  }

  static constexpr int NFRAG = NSPLIT * DT * KP;
  __device__ __forceinline__ void store_frags(Frag<T>* out) const {
    const int l = threadIdx.x % WAVE;
#pragma unroll
    for (int sp = 0; sp < NSPLIT; ++sp)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int ks = 0; ks < KP; ++ks) out[((sp * DT + dt) * KP + ks) * WAVE + l] = w[sp][dt][ks];
  }
  __device__ __forceinline__ void load_frags(const Frag<T>* in) {
    const int l = threadIdx.x % WAVE;
#pragma unroll
    for (int sp = 0; sp < NSPLIT; ++sp)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int ks = 0; ks < KP; ++ks) w[sp][dt][ks] = in[((sp * DT + dt) * KP + ks) * WAVE + l];
  }
};

// Per-head frequency fragments prepared once per call: for each wave, the
// projection fragments (FreqSlice) followed by the dX fragments (WTSlice).
template <class T, int D, int FW, bool NS>
struct FragBlock {
  static constexpr int NP = FreqSlice<T, D, FW, NS>::NFRAG;
  static constexpr int NT_ = WTSlice<T, D, FW, NS>::NFRAG;
  static constexpr int PER_WAVE = (NP + NT_) * WAVE;   // fragments per wave
  __device__ static const Frag<T>* proj(const void* base, int h, int nw, int w) {
    return static_cast<const Frag<T>*>(base) + ((size_t)h * nw + w) * PER_WAVE;
  }
  __device__ static const Frag<T>* dx(const void* base, int h, int nw, int w) {
    return proj(base, h, nw, w) + NP * WAVE;
  }
};

// One wave per (head, wave slice, part): part 0 writes the projection
// fragments, part 1 (launched for the backward only) the dX fragments.
template <class T, int D, int FW, int NW, bool NS>
__device__ __forceinline__ void prep_freqs_part(const float* W1, const float* W2, void* out, int wstride,
                                                int h, int w, int part) {
  typedef FragBlock<T, D, FW, NS> FBk;
  const float* W1h = W1 + (size_t)h * wstride;
  const float* W2h = NS ? W2 + (size_t)h * wstride : nullptr;
  Frag<T>* base = static_cast<Frag<T>*>(out) + ((size_t)h * NW + w) * FBk::PER_WAVE;
  if (part == 0) {
    FreqSlice<T, D, FW, NS> fs;
    fs.load(W1h, W2h, w * FW);
    fs.store_frags(base);
  } else {
    WTSlice<T, D, FW, NS> wt;
    wt.load(W1h, W2h, w * FW);
    wt.store_frags(base + FBk::NP * WAVE);
  }
}
// Grid (H, NW, parts), 64 threads.
template <class T, int D, int FW, int NW, bool NS>
__global__ __launch_bounds__(WAVE) void k_prep_freqs(const float* W1, const float* W2, void* out, int wstride) {
  prep_freqs_part<T, D, FW, NW, NS>(W1, W2, out, wstride, blockIdx.x, blockIdx.y, blockIdx.z);
}
// Both parts for two wave splits A and B in one launch: grid (H, max(NWA,
// NWB), 4); blockIdx.z = 2 * split + part.
template <class T, int D, int FWA, int NWA, int FWB, int NWB, bool NS>
__global__ __launch_bounds__(WAVE) void k_prep_freqs2(const float* W1, const float* W2, void* outA, void* outB,
                                                      int wstride) {
  const int w = blockIdx.y, part = blockIdx.z % 2;
  if (blockIdx.z < 2) {
    if (w < NWA) prep_freqs_part<T, D, FWA, NWA, NS>(W1, W2, outA, wstride, blockIdx.x, w, part);
  } else {
    if (w < NWB) prep_freqs_part<T, D, FWB, NWB, NS>(W1, W2, outB, wstride, blockIdx.x, w, part);
  }
}




// Trigonometric values of a projection in revolutions: cos(2 pi p), sin(2 pi p).
// v_sin_f32 / v_cos_f32 take revolutions and reduce the argument themselves:
// measured on gfx950 over |p| <= 200 their absolute error is 1.25e-7, lower
// than after an explicit v_fract_f32 (2.6e-7), so no reduction is done here.
__device__ __forceinline__ void sincos_rev(float p, float& s, float& c) {
  s = __builtin_amdgcn_sinf(p);
  c = __builtin_amdgcn_cosf(p);
}
__device__ __forceinline__ float cos_rev(float p) { return __builtin_amdgcn_cosf(p); }
// fp32 path: a float64 phase in revolutions.  r = p - rint(p) is exact in
// float64 and lies in [-1/2, 1/2].  It is split as r = rh + rl with rh its
// fp32 rounding (|rl| <= 2^-26); sine and cosine of rh come from v_sin_f32 /
// v_cos_f32 and the remainder enters to first order:
// sin 2pi(rh + rl) = sin 2pi rh + 2pi rl cos 2pi rh + O(rl^2).
__device__ __forceinline__ void sincos_rev(double p, float& s, float& c) {
  const double r = p - rint(p);
  const float rh = (float)r;
  const float a = 6.2831853f * (float)(r - (double)rh);
  const float s0 = __builtin_amdgcn_sinf(rh), c0 = __builtin_amdgcn_cosf(rh);
  s = fmaf(a, c0, s0);
  c = fmaf(-a, s0, c0);
}
__device__ __forceinline__ float cos_rev(double p) {
  const double r = p - rint(p);
  const float rh = (float)r;
  const float a = 6.2831853f * (float)(r - (double)rh);
  return fmaf(-a, __builtin_amdgcn_sinf(rh), __builtin_amdgcn_cosf(rh));
}

// Frequencies of wave w's slice (FW frequencies from w FW) that exist when
// the launch's group holds fvalid of its frequencies: the kernel variants
// compiled for a padded group (MASK) mask the rest; the others keep every
// feature, decided at compile time.
template <bool MASK, int FW>
__device__ __forceinline__ int slice_valid(int fvalid, int w) {
  if constexpr (!MASK) return FW;
  else return __builtin_amdgcn_readfirstlane(fvalid - w * FW);
}

// Zero the slots of an operand fragment of frequency tile ft (slots i and
// 4 + i: slice frequency ft*16 + 4g + i) whose frequency is not below fv.
template <class T>
__device__ __forceinline__ void mask_features(Frag<T>& f, int ft, int fv) {
  const int g = (threadIdx.x % WAVE) / 16;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (ft * 16 + 4 * g + i >= fv) { f.set(i, 0.0f); f.set(4 + i, 0.0f); }
}

// Feature epilogue for one frequency tile ft of one 16-token tile:
// scale = s * e(x) (0 for rows that are not valid).  Returns the operand
// fragment [cos-type features 4g..4g+3 | sin-type features 4g..4g+3].
// fv: frequencies of the wave's slice that exist (the last frequency group of
// an m that is not a multiple of the group width pads its slice with zero
// rows of W, whose features must vanish, not be cos 0 = 1): the features of
// slice frequencies ft*16 + 4g + i >= fv are zero.  The default keeps them all
// and compiles to the unmasked code.
template <class T, int FT, bool NS, class P>
__device__ __forceinline__ Frag<T> features(const P (&p)[NS ? 2 * FT : FT], int ft, float scale,
                                            int fv = FT * 16) {
  Frag<T> f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float s1, c1;
    sincos_rev(p[ft][i], s1, c1);
    const float sc = NS ? scale * cos_rev(p[FT + ft][i]) : scale;
    f.set(i, c1 * sc);
    f.set(4 + i, s1 * sc);
  }
  if (fv < FT * 16) mask_features(f, ft, fv);
  return f;
}

// Row scale s * exp(||x||^2 / exp(tau)) for valid rows, 0 otherwise.
__device__ __forceinline__ float row_scale(float ssq, float inv_c, float s_const, bool ok) {
  return ok ? s_const * __expf(ssq * inv_c) : 0.0f;
}
// fp32 path: the squared norm and 1/exp(tau) in float64, one rounding at the end.
__device__ __forceinline__ float row_scale(double ssq, double inv_c, float s_const, bool ok) {
  return ok ? (float)((double)s_const * exp(ssq * inv_c)) : 0.0f;
}
// 1 / exp(tau) in the precision of the path's norm factor.
template <class T> struct InvC {
  __device__ static __forceinline__ float of(float tau) { return __expf(-tau); }
};
template <> struct InvC<float> {
  __device__ static __forceinline__ double of(float tau) { return exp(-(double)tau); }
};
template <class T> __device__ __forceinline__ auto inv_c_of(float tau) { return InvC<T>::of(tau); }

}  // namespace flex
