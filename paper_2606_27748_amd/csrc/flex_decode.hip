// Recurrent decode step of the causal RFF linear attention: one new token per
// (b,h) slice against a running state (Eq.(linear att) restricted to j <= t,
// evaluated as the prefix state S'_t = S'_{t-1} + phi(k_t) [v_t ; 1]^T).
//
//   state  [BH][2m][dv+1] fp32, features in [cos | sin] order (Eq.(phi_n) /
//          Eq.(phi_non)), the last column the normaliser z = sum phi(k)
//   O_t    = (phi(q_t)^T S'_t)[:dv] / (phi(q_t)^T z_t),  den_t = phi(q_t)^T z_t
//
// One workgroup per slice.  The new token's projections and features are
// computed in fp32 from the fp32 frequencies (no operand rounding); the
// state is updated in place and read out in the same pass.  The state
// read-modify-write dominates: the step is bound by HBM bandwidth.
#include "flex_common.hpp"
#include "flex_kernels.hpp"

namespace flex {

namespace {
constexpr int DEC_NT = 256;   // threads per workgroup
}

template <class IO>
__global__ __launch_bounds__(DEC_NT) void k_decode_step(DecodeArgs a) {
  extern __shared__ float sm[];
  const int bh = blockIdx.x, h = bh % a.H, t = threadIdx.x;
  const int d = a.d, dv = a.dv, m = a.m, F = 2 * m, C = dv + 1;
  float* xq = sm;              // [d]
  float* xk = xq + d;          // [d]
  float* xv = xk + d;          // [dv + 1], last entry 1
  float* fq = xv + C;          // [F] phi(q)
  float* fk = fq + F;          // [F] phi(k)
  float* red = fk + F;         // [2] squared norms, then [R][C] readout partials

  const IO* q = static_cast<const IO*>(a.q) + (size_t)bh * d;
  const IO* k = static_cast<const IO*>(a.k) + (size_t)bh * d;
  const IO* v = static_cast<const IO*>(a.v) + (size_t)bh * dv;
  for (int i = t; i < d; i += DEC_NT) {
    xq[i] = io_to_float(q[i]);
    xk[i] = io_to_float(k[i]);
  }
  for (int i = t; i < dv; i += DEC_NT) xv[i] = io_to_float(v[i]);
  if (t == 0) xv[dv] = 1.0f;
  __syncthreads();
  // squared norms in a fixed order (one wave, lane-strided then a DPP tree)
  if (t < WAVE) {
    float sq = 0.f, sk = 0.f;
    for (int i = t; i < d; i += WAVE) {
      sq += xq[i] * xq[i];
      sk += xk[i] * xk[i];
    }
    sq = group_sum(lane_sum<16>(sq));
    sk = group_sum(lane_sum<16>(sk));
    if (t == 0) { red[0] = sq; red[1] = sk; }
  }
  __syncthreads();
  const float inv_c = __expf(-a.tau[h]);
  const float scq = a.s_const * __expf(red[0] * inv_c);
  const float sck = a.s_const * __expf(red[1] * inv_c);
  __syncthreads();   // red[] is reused below

  // projections and features, one frequency per thread and pass
  const float* W1 = a.W1 + (size_t)h * m * d;
  const float* W2 = a.W2 ? a.W2 + (size_t)h * m * d : nullptr;
  for (int f = t; f < m; f += DEC_NT) {
    float p1q = 0.f, p1k = 0.f, p2q = 0.f, p2k = 0.f;
    const float4* r1 = reinterpret_cast<const float4*>(W1 + (size_t)f * d);
    const float4* r2 = W2 ? reinterpret_cast<const float4*>(W2 + (size_t)f * d) : nullptr;
    for (int i4 = 0; i4 < d / 4; ++i4) {
      const float4 w1 = r1[i4];
      const float w1v[4] = {w1.x, w1.y, w1.z, w1.w};
      float w2v[4] = {0.f, 0.f, 0.f, 0.f};
      if (r2) {
        const float4 w2 = r2[i4];
        w2v[0] = w2.x; w2v[1] = w2.y; w2v[2] = w2.z; w2v[3] = w2.w;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = 4 * i4 + j;
        if (r2) {
          const float a1 = 0.5f * (w1v[j] + w2v[j]), a2 = 0.5f * (w1v[j] - w2v[j]);   // omega'_1, omega'_2
          p1q += a1 * xq[i]; p1k += a1 * xk[i];
          p2q += a2 * xq[i]; p2k += a2 * xk[i];
        } else {
          p1q += w1v[j] * xq[i]; p1k += w1v[j] * xk[i];
        }
      }
    }
    float sq1, cq1, sk1, ck1;
    sincos_rev(p1q * INV_2PI, sq1, cq1);
    sincos_rev(p1k * INV_2PI, sk1, ck1);
    const float mq = W2 ? scq * cos_rev(p2q * INV_2PI) : scq;
    const float mk = W2 ? sck * cos_rev(p2k * INV_2PI) : sck;
    fq[f] = cq1 * mq; fq[m + f] = sq1 * mq;
    fk[f] = ck1 * mk; fk[m + f] = sk1 * mk;
  }
  __syncthreads();

  // state update and readout: R groups of C threads, group r takes rows
  // f = r, r + R, ...; thread (r, c) owns column c of those rows
  const int R = DEC_NT / C;
  const int r = t / C, c = t % C;
  float acc = 0.f;
  if (r < R) {
    float* S = a.state + (size_t)bh * F * C + c;
    const float vc = xv[c];
#pragma unroll 8
    for (int f = r; f < F; f += R) {
      const float s = S[(size_t)f * C] + fk[f] * vc;
      S[(size_t)f * C] = s;
      acc += fq[f] * s;
    }
    red[r * C + c] = acc;
  }
  __syncthreads();
  // fixed-order sum over the groups; the normaliser column gives den
  if (t < C) {
    float s = 0.f;
    for (int g = 0; g < R; ++g) s += red[g * C + t];
    red[R * C + t] = s;
  }
  __syncthreads();
  if (t < dv) {
    const float dn = red[R * C + dv];
    IO* o = static_cast<IO*>(a.o) + (size_t)bh * dv;
    o[t] = float_to_io<IO>(red[R * C + t] / dn);
    if (a.den && t == 0) a.den[bh] = dn;
  }
}

size_t decode_smem_bytes(int d, int dv, int m) {
  const int C = dv + 1, R = DEC_NT / C;
  return (size_t)(2 * d + C + 4 * m + 2 + (R + 1) * C) * sizeof(float);
}

hipError_t launch_decode(const DecodeArgs& a, bool bf16, hipStream_t st) {
  const size_t smem = decode_smem_bytes(a.d, a.dv, a.m);
  if (bf16)
    k_decode_step<u16><<<a.BH, DEC_NT, smem, st>>>(a);
  else
    k_decode_step<float><<<a.BH, DEC_NT, smem, st>>>(a);
  return hipGetLastError();
}

}  // namespace flex
