// Recurrent decode step of the causal RFF linear attention: one new token per
// (b,h) slice against a running state (Eq.(linear att) restricted to j <= t,
// evaluated as the prefix state S'_t = S'_{t-1} + phi(k_t) [v_t ; 1]^T).
//
//   state  per slice: S [2m][dv] fp32, then z [2m] fp32 (the normaliser
//          column of S'); feature rows in [cos | sin] order (Eq.(phi_n) /
//          Eq.(phi_non))
//   O_t    = (phi(q_t)^T S_t) / (phi(q_t)^T z_t),  den_t = phi(q_t)^T z_t
//
// One workgroup per slice.  The new token's projections and features are
// computed in fp32 from the fp32 frequencies (no operand rounding); the
// state is updated in place and read out in the same pass.  The state
// read-modify-write dominates: the step is bound by HBM bandwidth, so S rows
// move as 16-byte lanes and the first rows are requested before the features
// are computed.
#include "flex_common.hpp"
#include "flex_kernels.hpp"

namespace flex {

namespace {
constexpr int DEC_NT = 256;   // threads per workgroup
constexpr int DEC_RB = 8;     // S rows (16-byte chunks) per thread and register batch
constexpr int DEC_ZR = 8;     // z entries per thread: 2m <= DEC_NT * DEC_ZR
constexpr int BUF_FLAGS = 0x00020000;   // raw dword buffer (CDNA descriptor word 3)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Loads one register batch of S: rows f = g + RG*(b*DEC_RB + j), j < cnt, at
// the lane's 16-byte column chunk.  The lane offset is one VGPR and the row
// step a scalar offset; the lanes of a wave read whole consecutive rows.
__device__ __forceinline__ void load_rows(float4 (&buf)[DEC_RB], __amdgpu_buffer_rsrc_t rs,
                                          int voff, int b, int cnt, int row_bytes) {
#pragma unroll
  for (int j = 0; j < DEC_RB; ++j)
    if (j < cnt)
      buf[j] = __builtin_bit_cast(
          float4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, (b * DEC_RB + j) * row_bytes, 0));
}
}  // namespace

template <class IO>
__global__ __launch_bounds__(DEC_NT) __attribute__((amdgpu_waves_per_eu(4))) void k_decode_step(
    DecodeArgs a) {
  extern __shared__ float4 sm4[];   // 16-byte aligned: x rows and readout partials are float4
  float* sm = reinterpret_cast<float*>(sm4);
  const int bh = blockIdx.x, h = bh % a.H, t = threadIdx.x;
  const int d = a.d, dv = a.dv, m = a.m, F = 2 * m;
  const int C4 = dv / 4, RG = DEC_NT / C4;   // column chunks per row, row groups
  float* xq = sm;              // [d]
  float* xk = xq + d;          // [d]
  float* xv = xk + d;          // [dv]
  float* red = xv + dv;        // [RG][dv] readout partials
  float* zred = red + RG * dv; // [DEC_NT / WAVE] normaliser partials, then [2] squared norms
  float* fq = zred + DEC_NT / WAVE + 4;   // [F] phi(q)
  float* fk = fq + F;          // [F] phi(k)

  // S pass geometry: lane (g, cc) owns column chunk cc of rows f = g, g + RG, ...
  const int g = t / C4, cc = t % C4;
  const int nrows = g < RG ? (F - g + RG - 1) / RG : 0;
  const int nbatch = (nrows + DEC_RB - 1) / DEC_RB;
  float* S = a.state + (size_t)bh * F * (dv + 1);
  float* z = S + (size_t)F * dv;
  // one slice's S block as a buffer resource: an access beyond its extent
  // would read zero and drop the store
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(S, 0, F * dv * (int)sizeof(float), BUF_FLAGS);
  const int voff = (g * dv + 4 * cc) * (int)sizeof(float);
  const int row_bytes = RG * dv * (int)sizeof(float);
  float4 cur[DEC_RB], nxt[DEC_RB];
  load_rows(cur, rs, voff, 0, min(nrows, DEC_RB), row_bytes);
  float zv[DEC_ZR];
#pragma unroll
  for (int j = 0; j < DEC_ZR; ++j)
    if (t + j * DEC_NT < F) zv[j] = z[t + j * DEC_NT];

  const IO* q = static_cast<const IO*>(a.q) + (size_t)bh * d;
  const IO* k = static_cast<const IO*>(a.k) + (size_t)bh * d;
  const IO* v = static_cast<const IO*>(a.v) + (size_t)bh * dv;
  for (int i = t; i < d; i += DEC_NT) {
    xq[i] = io_to_float(q[i]);
    xk[i] = io_to_float(k[i]);
  }
  for (int i = t; i < dv; i += DEC_NT) xv[i] = io_to_float(v[i]);
  __syncthreads();
  // squared norms in a fixed order (one wave, lane-strided then a DPP tree)
  float* nrm = zred + DEC_NT / WAVE;
  if (t < WAVE) {
    float sq = 0.f, sk = 0.f;
    for (int i = t; i < d; i += WAVE) {
      sq += xq[i] * xq[i];
      sk += xk[i] * xk[i];
    }
    sq = group_sum(lane_sum<16>(sq));
    sk = group_sum(lane_sum<16>(sk));
    if (t == 0) { nrm[0] = sq; nrm[1] = sk; }
  }
  __syncthreads();
  const float inv_c = __expf(-a.tau[h]);
  const float scq = a.s_const * __expf(nrm[0] * inv_c);
  const float sck = a.s_const * __expf(nrm[1] * inv_c);

  // projections and features: four adjacent lanes per frequency, lane u
  // takes the float4 chunks u, u + 4, ... of the frequency rows (the four
  // lanes read 64 consecutive bytes), a butterfly combines the partial dot
  // products, lane 0 writes phi(q) and lane 1 phi(k)
  const float* W1 = a.W1 + (size_t)h * m * d;
  const float* W2 = a.W2 ? a.W2 + (size_t)h * m * d : nullptr;
  const int u = t & 3, d4 = d / 4;
  const float4* xq4 = reinterpret_cast<const float4*>(xq);
  const float4* xk4 = reinterpret_cast<const float4*>(xk);
  for (int f0 = 0; f0 < m; f0 += DEC_NT / 4) {
    const int f = f0 + (t >> 2);
    float p1q = 0.f, p1k = 0.f, p2q = 0.f, p2k = 0.f;
    if (f < m) {
      const float4* r1 = reinterpret_cast<const float4*>(W1 + (size_t)f * d);
      const float4* r2 = W2 ? reinterpret_cast<const float4*>(W2 + (size_t)f * d) : nullptr;
#pragma unroll 4
      for (int i4 = u; i4 < d4; i4 += 4) {
        const float4 w1 = r1[i4], vq = xq4[i4], vk = xk4[i4];
        if (r2) {
          const float4 w2 = r2[i4];
          // omega'_1 = (w1 + w2) / 2, omega'_2 = (w1 - w2) / 2
          const float4 a1 = make_float4(0.5f * (w1.x + w2.x), 0.5f * (w1.y + w2.y),
                                        0.5f * (w1.z + w2.z), 0.5f * (w1.w + w2.w));
          const float4 a2 = make_float4(0.5f * (w1.x - w2.x), 0.5f * (w1.y - w2.y),
                                        0.5f * (w1.z - w2.z), 0.5f * (w1.w - w2.w));
          p1q += a1.x * vq.x + a1.y * vq.y + a1.z * vq.z + a1.w * vq.w;
          p1k += a1.x * vk.x + a1.y * vk.y + a1.z * vk.z + a1.w * vk.w;
          p2q += a2.x * vq.x + a2.y * vq.y + a2.z * vq.z + a2.w * vq.w;
          p2k += a2.x * vk.x + a2.y * vk.y + a2.z * vk.z + a2.w * vk.w;
        } else {
          p1q += w1.x * vq.x + w1.y * vq.y + w1.z * vq.z + w1.w * vq.w;
          p1k += w1.x * vk.x + w1.y * vk.y + w1.z * vk.z + w1.w * vk.w;
        }
      }
    }
#pragma unroll
    for (int o = 1; o < 4; o <<= 1) {
      p1q += __shfl_xor(p1q, o, 4);
      p1k += __shfl_xor(p1k, o, 4);
      p2q += __shfl_xor(p2q, o, 4);
      p2k += __shfl_xor(p2k, o, 4);
    }
    if (f < m && u < 2) {
      const float p1 = u == 0 ? p1q : p1k, p2 = u == 0 ? p2q : p2k;
      const float sc = u == 0 ? scq : sck;
      float s1, c1;
      sincos_rev(p1 * INV_2PI, s1, c1);
      const float mg = W2 ? sc * cos_rev(p2 * INV_2PI) : sc;
      float* fo = u == 0 ? fq : fk;
      fo[f] = c1 * mg;
      fo[m + f] = s1 * mg;
    }
  }
  __syncthreads();

  // S update and readout, one register batch at a time; the next batch is
  // requested before the current one is consumed
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (g < RG) {
    const float4 vc = reinterpret_cast<const float4*>(xv)[cc];
    for (int b = 0; b < nbatch; ++b) {
      const int cnt = min(nrows - b * DEC_RB, DEC_RB);
      if (b + 1 < nbatch)
        load_rows(nxt, rs, voff, b + 1, min(nrows - (b + 1) * DEC_RB, DEC_RB), row_bytes);
#pragma unroll
      for (int j = 0; j < DEC_RB; ++j) {
        if (j < cnt) {
          const int f = g + RG * (b * DEC_RB + j);
          const float kf = fk[f], qf = fq[f];
          float4 s4 = cur[j];
          s4.x += kf * vc.x; s4.y += kf * vc.y; s4.z += kf * vc.z; s4.w += kf * vc.w;
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, s4), rs, voff,
                                                 (b * DEC_RB + j) * row_bytes, 0);
          acc.x += qf * s4.x; acc.y += qf * s4.y; acc.z += qf * s4.z; acc.w += qf * s4.w;
        }
      }
#pragma unroll
      for (int j = 0; j < DEC_RB; ++j) cur[j] = nxt[j];
    }
    reinterpret_cast<float4*>(red)[g * C4 + cc] = acc;
  }
  // z update and its readout (the denominator), lane-strided then a fixed tree
  float dz = 0.f;
#pragma unroll
  for (int j = 0; j < DEC_ZR; ++j) {
    const int f = t + j * DEC_NT;
    if (f < F) {
      const float zn = zv[j] + fk[f];
      z[f] = zn;
      dz += fq[f] * zn;
    }
  }
  dz = group_sum(lane_sum<16>(dz));
  if ((t & (WAVE - 1)) == 0) zred[t / WAVE] = dz;
  __syncthreads();
  // fixed-order sums over the row groups and the waves
  if (t < dv) {
    float num = 0.f, dn = 0.f;
    for (int r = 0; r < RG; ++r) num += red[r * dv + t];
    for (int w = 0; w < DEC_NT / WAVE; ++w) dn += zred[w];
    IO* o = static_cast<IO*>(a.o) + (size_t)bh * dv;
    o[t] = float_to_io<IO>(num / dn);
    if (a.den && t == 0) a.den[bh] = dn;
  }
}

size_t decode_smem_bytes(int d, int dv, int m) {
  const int RG = DEC_NT / (dv / 4);
  return (size_t)(2 * d + dv + RG * dv + DEC_NT / WAVE + 4 + 4 * m) * sizeof(float);
}

hipError_t launch_decode(const DecodeArgs& a, bool bf16, hipStream_t st) {
  const size_t smem = decode_smem_bytes(a.d, a.dv, a.m);
  timing_mark(KC_DECODE, st, true);
  if (bf16)
    k_decode_step<u16><<<a.BH, DEC_NT, smem, st>>>(a);
  else
    k_decode_step<float><<<a.BH, DEC_NT, smem, st>>>(a);
  timing_mark(KC_DECODE, st, false);
  return hipGetLastError();
}

}  // namespace flex
