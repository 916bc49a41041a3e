// Attention-weight distillation loss L_awd (App. A.3; Sec. 4.3 distils softmax
// attention into the learnable kernel with it) and its gradient with respect
// to the kernel parameters W1, W2 and tau.  For every (b,h) slice, with the
// row softmax P = softmax(Q K^T / sqrt(d)) as the target and the kernel's
// weights A_ij = phi(Q_i)^T phi(K_j):
//
//   L         = -(1/N) sum_i sum_j P_ij log(A_ij / den_i),   den_i = sum_l A_il
//   G_ij      = dL/dA_ij = (1/N) (1/den_i - P_ij / A_ij)       (sum_j P_ij = 1)
//   dphi(Q_i) = sum_j G_ij phi(K_j),   dphi(K_j) = sum_i G_ij phi(Q_i)
//
// then the feature-map chain rule into dW'1, dW'2 (or dW) and dtau.  The N x N
// matrices never reach HBM: the quadratic passes stream 64-row tiles of one
// side through LDS against 16 rows per wave of the other side, form the logit
// tile Q K^T and the kernel tile phi phi^T on MFMA, and keep per-row
// statistics only.
//
//   k_awd_colsum  z = sum_j phi(K_j) per slice, so that den_i = phi(Q_i)^T z
//   k_awd_fwd     per 64-query tile: online base-2 log-sum-exp of the scaled
//                 logits and the P-weighted sum of log2(A_ij / den_i) per
//                 query; a loss partial per tile, (lse, 1/den) per query; with
//                 gradients also dphi(Q) in the same sweep
//   k_awd_bwd_k   dphi(K) per 64-key tile, streaming the query tiles
//   k_awd_wgrad   chain rule through phi for the Q and K rows of one head:
//                 dW' and dtau partials
//   k_awd_reduce  fixed-order sums into loss [B,H], dW1, dW2 and dtau
//
// Tile orientation of the quadratic passes: accumulator tiles have rows = the
// streamed side (4g + i) and columns = the wave's own rows (lane % 16).  When
// the queries are the own side, a query's statistics stay in one lane; a pair
// of such tiles is an operand over the streamed side with no transpose.
#include "flex_common.hpp"
#include "flex_stage.hpp"
#include "flex_kernels.hpp"

namespace flex {

namespace {
constexpr int AWD_NT = 256;   // threads of the quadratic passes: 4 waves x 16 own rows
constexpr int AWD_TILE = 64;  // rows of a tile on either side
constexpr float LN2 = 0.69314718055994531f;

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_fast(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float rcp_fast(float x) { return __builtin_amdgcn_rcpf(x); }

// Waves per SIMD the quadratic passes are compiled for: the bf16 shapes with
// up to 128 features fit 3 (4 for the d = 64 loss pass) without spilling; the
// others keep the compiler's choice.
template <class T, int D, int F, bool GRAD>
struct AwdOcc {
  static constexpr int value = (IsBf16<T>::value && F <= 128) ? ((GRAD || D < 64) ? 3 : 4) : 1;
};

// Operand fragments of one row (COLS columns, k = columns) of a row-major
// [N][COLS] io block; rows past the end read as zero.
template <class T, int COLS>
__device__ __forceinline__ void own_frags(Frag<T> (&f)[COLS / 32], const typename Io<T>::type* rows,
                                          int row, bool ok) {
  const int g = (threadIdx.x % WAVE) / 16;
#pragma unroll
  for (int ks = 0; ks < COLS / 32; ++ks) load8(f[ks], rows + (size_t)row * COLS + ks * 32 + 8 * g, ok);
}

// Logit and kernel tiles of the four 16-row blocks of the streamed tile:
// s[sub] = X_tile . x_own^T and a[sub] = Phi_tile . phi_own^T, rows = streamed
// rows sub*16 + 4g + i, columns = own rows.
template <class T, int D, int F, int LDX, int LDP>
__device__ __forceinline__ void tile_products(const typename Io<T>::type* XL, const typename Io<T>::type* PL,
                                              const Frag<T> (&xf)[D / 32], const Frag<T> (&pf)[F / 32],
                                              f32x4 (&s)[4], f32x4 (&a)[4]) {
  const int l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
#pragma unroll
  for (int sub = 0; sub < 4; ++sub) {
    s[sub] = zero4();
    a[sub] = zero4();
    const typename Io<T>::type* xrow = XL + (sub * 16 + r) * LDX;
    const typename Io<T>::type* prow = PL + (sub * 16 + r) * LDP;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      Frag<T> o;
      lds_row8(o, xrow, ks * 32 + 8 * g);
      mma(s[sub], o, xf[ks]);
    }
#pragma unroll
    for (int ks = 0; ks < F / 32; ++ks) {
      Frag<T> o;
      lds_row8(o, prow, ks * 32 + 8 * g);
      mma(a[sub], o, pf[ks]);
    }
  }
}

// Two accumulator tiles as one operand fragment split into a high and a low
// part (bf16 hi + lo carries about 16 significant bits; fp32 keeps the value).
template <class T>
__device__ __forceinline__ void split_pair(const f32x4& a, const f32x4& b, Frag<T>& hi, Frag<T>& lo) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hi.set(i, a[i]);
    hi.set(4 + i, b[i]);
    lo.set(i, a[i] - hi.get(i));
    lo.set(4 + i, b[i] - hi.get(4 + i));
  }
}
}  // namespace

// z[bh][f] = sum_j phi(K_j)_f in a fixed order: 16-byte column vectors per
// thread, row groups summed through LDS.
template <class IO, int F>
__global__ __launch_bounds__(256) void k_awd_colsum(const IO* __restrict__ phk, float* __restrict__ z, int N) {
  constexpr int VEC = 16 / sizeof(IO), CG = F / VEC, RG = 256 / CG;
  __shared__ float red[RG][F];
  const int bh = blockIdx.x, t = threadIdx.x, cg = t % CG, rg = t / CG;
  const IO* P = phk + (size_t)bh * N * F + cg * VEC;
  float acc[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
#pragma unroll 4
  for (int n = rg; n < N; n += RG) {
    const uint4 v = *reinterpret_cast<const uint4*>(P + (size_t)n * F);
    const IO* e = reinterpret_cast<const IO*>(&v);
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] += io_to_float(e[j]);
  }
#pragma unroll
  for (int j = 0; j < VEC; ++j) red[rg][cg * VEC + j] = acc[j];
  __syncthreads();
  for (int f = t; f < F; f += 256) {
    float s = 0.f;
#pragma unroll
    for (int g = 0; g < RG; ++g) s += red[g][f];
    z[(size_t)bh * F + f] = s;
  }
}

// Loss pass: one workgroup per (b,h, 64-query tile); wave w owns queries
// tile*64 + 16w + (lane % 16).  The four lane groups of a query share one
// running maximum of its scaled logits (a cross-group max per key tile); each
// lane sums 2^(x - max) (Z) and 2^(x - max) log2(A/den) (LS) over its own keys
// (4g + i of every 16-key block), merged at the end.
//
// DPHI also forms dphi(Q) in the same sweep (flash style):
//   dphi(Q_i) = (1/N) (z / den_i - U_i / Z_i),  U_i = sum_j 2^(x_ij - max) / A_ij phi(K_j),
// with U rescaled whenever the maximum grows.  The two terms cancel to the
// extent the kernel's weights match the target, so e/A enters the MFMA as a
// bf16 hi + lo pair (about 16 bits), not rounded to bf16.
template <class T, int D, int F, bool DPHI>
__global__ __launch_bounds__(AWD_NT) __attribute__((amdgpu_waves_per_eu(AwdOcc<T, D, F, DPHI>::value)))
void k_awd_fwd(AwdArgs a) {
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, AWD_NT> StX;
  typedef RowStage<IO, F, AWD_NT> StP;
  __shared__ __align__(16) IO XL[StX::LDS_ELEMS];
  __shared__ __align__(16) IO PL[StP::LDS_ELEMS];
  __shared__ float LP[AWD_NT / 4];
  const WgCoord wc = wg_coord(a.ntile, a.H, a.BH);
  const int tile = wc.seg, bh = wc.bh;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const IO* Q = static_cast<const IO*>(a.Q) + (size_t)bh * a.N * D;
  const IO* K = static_cast<const IO*>(a.K) + (size_t)bh * a.N * D;
  const IO* PQ = static_cast<const IO*>(a.phq) + (size_t)bh * a.N * F;
  const IO* PK = static_cast<const IO*>(a.phk) + (size_t)bh * a.N * F;
  const int q = tile * AWD_TILE + w * 16 + r;
  const bool qok = q < a.N;
  Frag<T> xf[D / 32], pf[F / 32];
  own_frags<T, D>(xf, Q, q, qok);
  own_frags<T, F>(pf, PQ, q, qok);
  // den_q = phi(Q_q)^T z (the row sum of A, from the column sums of phi(K))
  const float* z = a.z + (size_t)bh * F;
  float dp = 0.f;
#pragma unroll
  for (int ks = 0; ks < F / 32; ++ks)
#pragma unroll
    for (int j = 0; j < 8; ++j) dp += pf[ks].get(j) * z[ks * 32 + 8 * g + j];
  const float den = group_sum(dp);
  const float rden = 1.0f / den;

  float mx = -INFINITY, Z = 0.f, LS = 0.f;
  f32x4 U[DPHI ? F / 16 : 1];
#pragma unroll
  for (int ft = 0; ft < (DPHI ? F / 16 : 1); ++ft) U[ft] = zero4();
  StX sx;
  StP sp;
  sx.fetch(K, 0, a.N);
  sp.fetch(PK, 0, a.N);
  for (int kt = 0; kt < a.ntile; ++kt) {
    __syncthreads();   // the previous tile's LDS reads are done
    sx.store(XL);
    sp.store(PL);
    __syncthreads();
    {
      const int n1 = (kt + 1 < a.ntile ? kt + 1 : kt) * AWD_TILE;   // the last tile refetches itself (unused)
      sx.fetch(K, n1, a.N);
      sp.fetch(PK, n1, a.N);
    }
    f32x4 s[4], av[4];
    tile_products<T, D, F, StX::LD, StP::LD>(XL, PL, xf, pf, s, av);
    const int kb = kt * AWD_TILE + 4 * g;
    // whole tiles (every tile but a ragged last one) skip the key masks
    const bool full = (kt + 1) * AWD_TILE <= a.N;
    // the query's maximum over this tile's valid keys, shared by its four
    // lane groups (c1 > 0 scales raw logits into base 2)
    float tmax = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 4; ++sub)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (full || kb + sub * 16 + i < a.N) tmax = fmaxf(tmax, s[sub][i]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    tmax *= a.c1;
    const float mn = fmaxf(mx, tmax);
    const float al = mn > mx ? exp2_fast(mx - mn) : 1.f;   // 0 while mx is -inf
    Z *= al;
    LS *= al;
    if (DPHI && __any(al != 1.f)) {
      // rows 4g + i of U belong to queries 4g + i, whose factors sit in lanes 4g + i
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float ai = __shfl(al, 4 * g + i);
#pragma unroll
        for (int ft = 0; ft < (DPHI ? F / 16 : 1); ++ft) U[ft][i] *= ai;
      }
    }
    mx = mn;
    const float nm = -mx;
    f32x4 H[DPHI ? 4 : 1];
#pragma unroll
    for (int sub = 0; sub < 4; ++sub)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = full || kb + sub * 16 + i < a.N;
        const float e = ok ? exp2_fast(fmaf(s[sub][i], a.c1, nm)) : 0.f;
        Z += e;
        if (ok) LS = fmaf(e, log2_fast(av[sub][i] * rden), LS);
        if (DPHI) H[sub][i] = ok ? e * rcp_fast(av[sub][i]) : 0.f;
      }
    if (DPHI) {
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        Frag<T> hi, lo;
        split_pair<T>(H[2 * kp], H[2 * kp + 1], hi, lo);
#pragma unroll
        for (int ft = 0; ft < F / 16; ++ft) {
          const Frag<T> pb = lds_tr_frag<T>(reinterpret_cast<const T*>(PL), StP::LD, 32 * kp + 4 * g,
                                            32 * kp + 16 + 4 * g, ft * 16);
          mma(U[ft], hi, pb);
          if (IsBf16<T>::value) mma(U[ft], lo, pb);
        }
      }
    }
  }
  // the four lane groups of a query share its maximum: plain sums
  Z += __shfl_xor(Z, 16);
  Z += __shfl_xor(Z, 32);
  LS += __shfl_xor(LS, 16);
  LS += __shfl_xor(LS, 32);
  if (g == 0) {
    if (qok)
      reinterpret_cast<float2*>(a.stats)[(size_t)bh * a.N + q] =
          make_float2(mx + log2_fast(Z) + a.log2n, rden * a.inv_n);
    LP[w * 16 + r] = qok ? -LN2 * LS / Z : 0.f;
  }
  if (DPHI) {
    IO* dst = static_cast<IO*>(a.dphq) + (size_t)bh * a.N * F;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float zi = __shfl(Z, 4 * g + i), ri = __shfl(rden, 4 * g + i);
      const float iz = 1.0f / zi;
      const int row = tile * AWD_TILE + w * 16 + 4 * g + i;
#pragma unroll
      for (int ft = 0; ft < F / 16; ++ft) {
        const float v = a.inv_n * (ri * z[ft * 16 + r] - U[ft][i] * iz);
        if (row < a.N) dst[(size_t)row * F + ft * 16 + r] = float_to_io<IO>(v);
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int i = 0; i < AWD_NT / 4; ++i) t += LP[i];
    a.lpart[(size_t)bh * a.ntile + tile] = t;
  }
}

// Key-side gradient pass: dphi(K) for a 64-key tile, streaming the query tiles
// with their statistics.  G = (1/N)(1/den - P/A) per pair, then
// dphi(K) += G^T . Phi(Q) on MFMA with the streamed features read through the
// transpose load.  (dphi(Q) comes out of the loss pass.)
template <class T, int D, int F>
__global__ __launch_bounds__(AWD_NT) __attribute__((amdgpu_waves_per_eu(AwdOcc<T, D, F, true>::value)))
void k_awd_bwd_k(AwdArgs a) {
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, AWD_NT> StX;
  typedef RowStage<IO, F, AWD_NT> StP;
  __shared__ __align__(16) IO XL[StX::LDS_ELEMS];
  __shared__ __align__(16) IO PL[StP::LDS_ELEMS];
  __shared__ float2 SL[AWD_TILE];
  const WgCoord wc = wg_coord(a.ntile, a.H, a.BH);
  const int tile = wc.seg, bh = wc.bh;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const size_t xo = (size_t)bh * a.N * D, po = (size_t)bh * a.N * F;
  const IO* Xown = static_cast<const IO*>(a.K) + xo;
  const IO* Pown = static_cast<const IO*>(a.phk) + po;
  const IO* Xoth = static_cast<const IO*>(a.Q) + xo;
  const IO* Poth = static_cast<const IO*>(a.phq) + po;
  const float2* stats = reinterpret_cast<const float2*>(a.stats) + (size_t)bh * a.N;
  const int o = tile * AWD_TILE + w * 16 + r;
  const bool ook = o < a.N;
  Frag<T> xf[D / 32], pf[F / 32];
  own_frags<T, D>(xf, Xown, o, ook);
  own_frags<T, F>(pf, Pown, o, ook);
  f32x4 acc[F / 16];
#pragma unroll
  for (int ft = 0; ft < F / 16; ++ft) acc[ft] = zero4();

  StX sx;
  StP sp;
  sx.fetch(Xoth, 0, a.N);
  sp.fetch(Poth, 0, a.N);
  // per-row statistics: loaded unconditionally from a clamped row, zeroed past N when stored
  bool sr_ok = (int)threadIdx.x < a.N;
  float2 sr = stats[min((int)threadIdx.x % AWD_TILE, a.N - 1)];
  for (int ot = 0; ot < a.ntile; ++ot) {
    __syncthreads();
    sx.store(XL);
    sp.store(PL);
    if (threadIdx.x < AWD_TILE) SL[threadIdx.x] = sr_ok ? sr : make_float2(0.f, 0.f);
    __syncthreads();
    {
      const int n1 = (ot + 1 < a.ntile ? ot + 1 : ot) * AWD_TILE;   // the last tile refetches itself (unused)
      sx.fetch(Xoth, n1, a.N);
      sp.fetch(Poth, n1, a.N);
      const int row = n1 + (int)threadIdx.x % AWD_TILE;
      sr_ok = row < a.N;
      sr = stats[min(row, a.N - 1)];
    }
    f32x4 s[4], av[4];
    tile_products<T, D, F, StX::LD, StP::LD>(XL, PL, xf, pf, s, av);
    const int ob = ot * AWD_TILE + 4 * g;
    f32x4 G[4];
#pragma unroll
    for (int sub = 0; sub < 4; ++sub)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 st = SL[sub * 16 + 4 * g + i];
        const float p = exp2_fast(s[sub][i] * a.c1 - st.x);
        const float gv = st.y - p * rcp_fast(av[sub][i]);
        G[sub][i] = (ook && ob + sub * 16 + i < a.N) ? gv : 0.f;
      }
#pragma unroll
    for (int kp = 0; kp < 2; ++kp) {
      const Frag<T> gf = pair_tiles<T>(G[2 * kp], G[2 * kp + 1]);
#pragma unroll
      for (int ft = 0; ft < F / 16; ++ft)
        mma(acc[ft], gf,
            lds_tr_frag<T>(reinterpret_cast<const T*>(PL), StP::LD, 32 * kp + 4 * g, 32 * kp + 16 + 4 * g,
                           ft * 16));
    }
  }
  // dphi is stored in the io dtype: its rounding (2^-9 relative on the bf16
  // path) is below that of the bf16 features the passes already use
  IO* dst = static_cast<IO*>(a.dphk) + po;
#pragma unroll
  for (int ft = 0; ft < F / 16; ++ft)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = tile * AWD_TILE + w * 16 + 4 * g + i;
      if (row < a.N) dst[(size_t)row * F + ft * 16 + r] = float_to_io<IO>(acc[ft][i]);
    }
}

// Chain rule through phi for the Q and K rows of one head.  Grid (H, parts);
// wave w owns frequencies 16w .. 16w+15; the workgroup walks its share of the
// head's 32-row chunks (Q rows of every batch, then K rows), recomputes the
// projections on MFMA (bf16 hi + lo frequencies), forms dP per radian
//   stationary    dP  = Phi_cos dPhi_sin - Phi_sin dPhi_cos
//   nonstationary dP1 = Phi_a dPhi_b - Phi_b dPhi_a,
//                 dP2 = -s e sin P2 (cos P1 dPhi_a + sin P1 dPhi_b)
// and accumulates dW'[f][:] += dP[:, f]^T X (hi + lo split of dP on MFMA) and,
// over the K rows, <phi, dphi> ||x||^2 for dtau = -that / exp(tau).  The Q rows
// add nothing to dtau: the loss depends on A_ij / sum_l A_il only, which no
// rescaling of phi(Q_i) changes, so <phi(Q_i), dphi(Q_i)> = 0 exactly (formed
// from rounded products it would be pure rounding noise).
template <class T, int D, int M, bool NS>
__global__ __launch_bounds__(M / 16 * WAVE) void k_awd_wgrad(AwdArgs a) {
  typedef typename Io<T>::type IO;
  constexpr int NW = M / 16, NT = NW * WAVE, F = 2 * M, ROWS = 32;
  typedef RowStage<IO, D, NT, ROWS> StX;
  typedef RowStage<IO, F, NT, ROWS> StD;
  typedef FreqSlice<T, D, 16, NS> FS;
  __shared__ __align__(16) IO XL[StX::LDS_ELEMS];
  __shared__ __align__(16) IO DL[StD::LDS_ELEMS];
  __shared__ typename StX::Ssq SSQ[ROWS];
  __shared__ float TRED[NW];
  const int h = blockIdx.x, part = blockIdx.y;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  FS fs;
  fs.load(a.W1 + (size_t)h * M * D, NS ? a.W2 + (size_t)h * M * D : nullptr, w * 16);
  const auto inv_c = inv_c_of<T>(a.tau[h]);
  const int nch = (a.N + ROWS - 1) / ROWS, per_side = a.B * nch, U = 2 * per_side;
  const int u0 = (int)((long long)U * part / a.parts), u1 = (int)((long long)U * (part + 1) / a.parts);
  f32x4 dw[FS::PR][D / 16];
#pragma unroll
  for (int pr = 0; pr < FS::PR; ++pr)
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) dw[pr][dt] = zero4();
  float gt = 0.f;
  // chunk u -> rows n0.. of side (0: Q, 1: K) of slice (b, h)
  auto rows_of = [&](int u, const IO*& X, const IO*& dph, int& n0, int& side) {
    side = u / per_side;
    const int rem = u % per_side, b = rem / nch;
    const size_t bh = (size_t)b * a.H + h;
    X = static_cast<const IO*>(side ? a.K : a.Q) + bh * a.N * D;
    dph = static_cast<const IO*>(side ? a.dphk : a.dphq) + bh * a.N * F;
    n0 = (rem % nch) * ROWS;
  };
  StX sx;
  StD sd;
  if (u0 < u1) {
    const IO* X;
    const IO* dph;
    int n0, side;
    rows_of(u0, X, dph, n0, side);
    sx.fetch(X, n0, a.N);
    sd.fetch(dph, n0, a.N);
  }
  for (int u = u0; u < u1; ++u) {
    const IO* X;
    const IO* dph;
    int n0, side;
    rows_of(u, X, dph, n0, side);
    const float gw = side ? 1.f : 0.f;   // dtau takes the K rows only
    __syncthreads();
    sx.store(XL, SSQ);
    sd.store(DL);
    __syncthreads();
    {
      const IO* Xn;
      const IO* dn;
      int nn, sn;
      rows_of(u + 1 < u1 ? u + 1 : u, Xn, dn, nn, sn);   // the last unit refetches itself (unused)
      sx.fetch(Xn, nn, a.N);
      sd.fetch(dn, nn, a.N);
    }
    f32x4 dp[2][FS::PR];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      ProjT<T> p[FS::PR];
      project_rows_lds<T, D, 16, NS, StX::LD>(fs, XL, tt, p);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tl = tt * 16 + 4 * g + i, tok = n0 + tl;
        const bool ok = tok < a.N;
        const auto ssq = SSQ[tl];
        const float sc = row_scale(ssq, inv_c, a.s_const, ok);
        const int f = w * 16 + r;
        // rows past the end were staged as zeros
        const float da = io_to_float(DL[tl * StD::LD + f]);
        const float db = io_to_float(DL[tl * StD::LD + M + f]);
        float s1, c1;
        sincos_rev(p[0][i], s1, c1);
        if (NS) {
          float s2, c2;
          sincos_rev(p[FS::PR - 1][i], s2, c2);
          const float pa = sc * c1 * c2, pb = sc * s1 * c2;
          dp[tt][0][i] = pa * db - pb * da;
          dp[tt][FS::PR - 1][i] = -sc * s2 * (c1 * da + s1 * db);
          gt += gw * (pa * da + pb * db) * ssq;
        } else {
          const float pa = sc * c1, pb = sc * s1;
          dp[tt][0][i] = pa * db - pb * da;
          gt += gw * (pa * da + pb * db) * ssq;
        }
      }
    }
    Frag<T> xt[D / 16];
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      xt[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XL), StX::LD, 4 * g, 16 + 4 * g, dt * 16);
#pragma unroll
    for (int pr = 0; pr < FS::PR; ++pr) {
      Frag<T> hi, lo;
      split_pair<T>(dp[0][pr], dp[1][pr], hi, lo);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        mma(dw[pr][dt], hi, xt[dt]);
        if (IsBf16<T>::value) mma(dw[pr][dt], lo, xt[dt]);
      }
    }
  }
  float* out = a.wpart + ((size_t)h * a.parts + part) * FS::PR * M * D;
#pragma unroll
  for (int pr = 0; pr < FS::PR; ++pr)
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) out[((size_t)pr * M + w * 16 + 4 * g + i) * D + dt * 16 + r] = dw[pr][dt][i];
  const float s = group_sum(lane_sum<16>(gt));
  if (l == 0) TRED[w] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int i = 0; i < NW; ++i) t += TRED[i];
    a.dtpart[(size_t)h * a.parts + part] = -inv_c * t;
  }
}

// Fixed-order sums: dW'1, dW'2 -> dW1 = (dW'1 + dW'2)/2, dW2 = (dW'1 - dW'2)/2
// (W'1 = (W1 + W2)/2, W'2 = (W1 - W2)/2); dtau; loss = (1/N) sum of the tile
// partials.  Grid (element blocks of 64, H): the four waves of a block take
// every fourth partial of the block's 64 elements, then combine in order.
constexpr int AWD_RED_E = 64;
template <bool NS>
__global__ __launch_bounds__(256) void k_awd_reduce(AwdArgs a, int M, int D) {
  __shared__ float R[2][4][AWD_RED_E];
  const int h = blockIdx.y, w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
  const int e = blockIdx.x * AWD_RED_E + l, MD = M * D, nmat = NS ? 2 : 1;
  if (a.dW1) {
    float x0 = 0.f, x1 = 0.f;
    if (e < MD) {
#pragma unroll 4
      for (int p = w; p < a.parts; p += 4) {
        const float* src = a.wpart + ((size_t)h * a.parts + p) * nmat * MD;
        x0 += src[e];
        if (NS) x1 += src[MD + e];
      }
    }
    R[0][w][l] = x0;
    R[1][w][l] = x1;
    __syncthreads();
    if (w == 0 && e < MD) {
      const float y0 = ((R[0][0][l] + R[0][1][l]) + R[0][2][l]) + R[0][3][l];
      if (NS) {
        const float y1 = ((R[1][0][l] + R[1][1][l]) + R[1][2][l]) + R[1][3][l];
        a.dW1[(size_t)h * MD + e] = 0.5f * (y0 + y1);
        a.dW2[(size_t)h * MD + e] = 0.5f * (y0 - y1);
      } else {
        a.dW1[(size_t)h * MD + e] = y0;
      }
    }
  }
  if (blockIdx.x != 0) return;
  if (a.dW1 && a.dtau && threadIdx.x == 0) {
    float t = 0.f;
    for (int p = 0; p < a.parts; ++p) t += a.dtpart[(size_t)h * a.parts + p];
    a.dtau[h] = t;
  }
  for (int b = threadIdx.x; b < a.B; b += 256) {
    const size_t bh = (size_t)b * a.H + h;
    float t = 0.f;
    for (int i = 0; i < a.ntile; ++i) t += a.lpart[bh * a.ntile + i];
    a.loss[bh] = t * a.inv_n;
  }
}

namespace {
template <class T, int D, int M>
hipError_t run_awd(const AwdArgs& a, bool ns, bool grads, hipStream_t st) {
  typedef typename Io<T>::type IO;
  constexpr int F = 2 * M;
  const int nwg = a.BH * a.ntile;
  k_awd_colsum<IO, F><<<a.BH, 256, 0, st>>>(static_cast<const IO*>(a.phk), a.z, a.N);
  timing_mark(KC_AWD_FWD, st, true);
  if (grads)
    k_awd_fwd<T, D, F, true><<<nwg, AWD_NT, 0, st>>>(a);   // loss and dphi(Q)
  else
    k_awd_fwd<T, D, F, false><<<nwg, AWD_NT, 0, st>>>(a);
  timing_mark(KC_AWD_FWD, st, false);
  if (grads) {
    timing_mark(KC_AWD_BWD_K, st, true);
    k_awd_bwd_k<T, D, F><<<nwg, AWD_NT, 0, st>>>(a);
    timing_mark(KC_AWD_BWD_K, st, false);
    const dim3 wg(a.H, a.parts);
    timing_mark(KC_AWD_WGRAD, st, true);
    if (ns)
      k_awd_wgrad<T, D, M, true><<<wg, M / 16 * WAVE, 0, st>>>(a);
    else
      k_awd_wgrad<T, D, M, false><<<wg, M / 16 * WAVE, 0, st>>>(a);
    timing_mark(KC_AWD_WGRAD, st, false);
  }
  const dim3 rg(grads ? (M * D + AWD_RED_E - 1) / AWD_RED_E : 1, a.H);
  if (ns)
    k_awd_reduce<true><<<rg, 256, 0, st>>>(a, M, D);
  else
    k_awd_reduce<false><<<rg, 256, 0, st>>>(a, M, D);
  return hipGetLastError();
}
}  // namespace

bool awd_shape_supported(bool bf16, int d, int m) {
  if (bf16) return (d == 32 && m == 64) || (d == 64 && m == 64) || (d == 64 && m == 128);
  return d == 32 && m == 64;
}

// Workgroups of the chain-rule pass per head: about 512 in all, at most one
// per 32-row chunk of the head.
int awd_parts(int B, int H, int N) {
  const long long chunks = 2LL * B * ((N + 31) / 32);
  long long p = (512 + H - 1) / H;
  if (p > chunks) p = chunks;
  return (int)(p < 1 ? 1 : p);
}

hipError_t launch_awd(const AwdArgs& a, const KernelShape& ks, bool grads, hipStream_t st) {
  const bool ns = ks.nonstationary;
  if (ks.bf16) {
    if (ks.d == 32 && ks.m == 64) return run_awd<__bf16, 32, 64>(a, ns, grads, st);
    if (ks.d == 64 && ks.m == 64) return run_awd<__bf16, 64, 64>(a, ns, grads, st);
    if (ks.d == 64 && ks.m == 128) return run_awd<__bf16, 64, 128>(a, ns, grads, st);
  } else if (ks.d == 32 && ks.m == 64) {
    return run_awd<float, 32, 64>(a, ns, grads, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace flex
