// Forward kernels of the RFF linear attention (Eq.(linear att), Sec. 2.2) with
// the Flexformer feature maps (Eq.(phi_n) / Eq.(phi_non), Sec. 3.1-3.2).
//
// Work decomposition.  A workgroup owns one (b,h) slice and one contiguous
// segment of 64-token chunks.  Its NW waves split the m frequencies: wave w
// owns frequencies [w*FW, (w+1)*FW), i.e. 2*FW of the d' = 2m features, and
// keeps its rows of the state S' = sum_j phi(K_j) [V_j ; 1]^T (d' x (dv+1),
// fp32) as MFMA accumulators.  Per chunk a wave forms phi(Q), phi(K) for its
// features on chip (projection + fused trig, never written to memory), adds
// its partial readout phi(Q) S' plus the intra-chunk masked term
// tril(phi(Q) phi(K)^T) [V;1], and the partials of the NW waves are summed in
// LDS before O = num / den is written.
//
// Causal sequences are split into segments for occupancy:
//   k_fwd_state  : segment-local states (one pass over K, V),
//   k_state_scan : exclusive prefix over segments (causal) or the total
//                  (non-causal), fixed order, deterministic,
//   k_fwd_sweep  : per segment, carry-in state + chunk sweep, writes O, den.
#include "flex_common.hpp"
#include "flex_kernels.hpp"
#include "flex_stage.hpp"

namespace flex {

// ---------------------------------------------------------------------------
// Segment-local state: S'_seg = sum over the segment's tokens of phi(K)[V;1]^T.
// ---------------------------------------------------------------------------
// MASK: the variant for a padded frequency group (features of its padding
// rows masked to zero), as in the sweeps.
template <class T, int D, int FW, int NW, bool NS, bool MASK = false>
__global__ __launch_bounds__(NW * WAVE) __attribute__((amdgpu_waves_per_eu(state_waves_per_eu(D, NS), state_waves_per_eu(D, NS))))
void k_fwd_state(FwdArgs a) {
  typedef Shape<T, D, FW, NW, NS> SH;
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, SH::NT> StK;
  typedef RowStage<IO, SH::DV, SH::NT> StV;
  __shared__ __attribute__((aligned(16))) IO XK[StK::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) float SCK[CHUNK];   // staged: per-token scale s e(k)
  __shared__ __attribute__((aligned(16))) IO XV[StV::LDS_ELEMS];   // [token][value col]

  const WgCoord wc = wg_coord(a.pre_segs * a.sub, a.H, a.BH);   // seg: sub-segment
  const int seg = wc.seg, bh = wc.bh, h = bh % a.H;
  const int w = threadIdx.x / WAVE;
  const int fv = slice_valid<MASK, FW>(a.fvalid, w);
  const int cps = a.chunks_per_seg / a.sub;
  const int c0 = seg * cps;
  const int c1 = min(c0 + cps, a.nchunks);
  const IO* K = static_cast<const IO*>(a.K) + (size_t)bh * a.N * D;
  const IO* V = static_cast<const IO*>(a.V) + (size_t)bh * a.N * SH::DV;

  StK sk;
  StV sv;
  if (c0 < c1) {
    sk.fetch(K, c0 * CHUNK, a.N);
    sv.fetch(V, c0 * CHUNK, a.N);
  }
  const Frag<T>* wproj = FragBlock<T, D, FW, NS>::proj(a.wfrag, h, NW, w);
  const auto inv_c = inv_c_of<T>(a.tau[h]);

  f32x4 S[SH::FC][SH::DVT1];
#pragma unroll
  for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt) S[fc][dt] = zero4();
  const Frag<T> ones = ones_col0<T>();
  const int g = (threadIdx.x % WAVE) / 16;

  // projection fragments: held for the whole sweep where registers allow
  // (d <= 64), else reloaded per chunk ahead of the staging barriers
  constexpr bool KEEP_FS = D <= 64;
  FreqSlice<T, D, FW, NS> fs;
  // held for the whole sweep: built from W by each wave (no prepared copy is needed)
  if (KEEP_FS) fs.load(a.W1 + (size_t)h * a.w_stride, NS ? a.W2 + (size_t)h * a.w_stride : nullptr, w * FW);
  for (int c = c0; c < c1; ++c) {
    const int tok0 = c * CHUNK;
    if (!KEEP_FS) fs.load_frags(wproj);
    __syncthreads();
    sk.store(XK, SCK, [&](int t, auto ssq) { return row_scale(ssq, inv_c, a.s_const, tok0 + t < a.N); });
    sv.store(XV);
    {
      const int t1 = c + 1 < c1 ? tok0 + CHUNK : tok0;   // the last chunk refetches itself (unused)
      sk.fetch(K, t1, a.N);
      sv.fetch(V, t1, a.N);
    }
    __syncthreads();
    // phi(K) with the tokens as the contraction index, straight from registers
#pragma unroll
    for (int ks = 0; ks < SH::KT; ++ks) {
      Frag<T> pk[SH::FC];
      feature_frags_rows<T, D, FW, NS, StK::LD>(fs, XK, SCK, ks, pk, fv);
      Frag<T> vf[SH::DVT];
#pragma unroll
      for (int dt = 0; dt < SH::DVT; ++dt) vf[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XV), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16);
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) {
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt) mma(S[fc][dt], pk[fc], vf[dt]);
        mma(S[fc][SH::DVT], pk[fc], ones);
      }
    }
  }
  float* out = a.state + ((size_t)bh * a.segments * a.sub + seg) * SH::STATE + (size_t)w * SH::WAVE_STATE;
  const int l = threadIdx.x % WAVE;
#pragma unroll
  for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
      *reinterpret_cast<f32x4*>(out + ((fc * SH::DVT1 + dt) * WAVE + l) * 4) = S[fc][dt];
}

// ---------------------------------------------------------------------------
// Exclusive prefix over segments (causal) or total into segment 0 (non-causal).
// state: [BH][P][E] fp32.  Fixed summation order.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_state_scan(float* state0, float* state1, int P, int sub, int E,
                                                    int causal, int reverse0, int nread0) {
  // one thread per 4 consecutive elements (E is a multiple of 256)
  const int e4 = blockIdx.x * 256 + threadIdx.x;
  if (4 * e4 >= E) return;
  const int n = P * sub;
  // blockIdx.z selects the state array: state0 in the direction reverse0,
  // state1 (backward only) in the opposite one
  const int reverse = blockIdx.z == 0 ? reverse0 : 1 - reverse0;
  float4* s = reinterpret_cast<float4*>((blockIdx.z == 0 ? state0 : state1) + (size_t)blockIdx.y * n * E) + e4;
  const size_t E4 = E / 4;
  const int nread = blockIdx.z == 0 ? nread0 : n;   // slots holding local states (scan order)
  constexpr int BATCH = 16;  // independent loads in flight per thread
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k0 = 0; k0 < n; k0 += BATCH) {
    float4 v[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int k = k0 + j;
      const int p = reverse ? n - 1 - k : k;
      v[j] = k < nread ? s[(size_t)p * E4] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (causal) {
#pragma unroll
      for (int j = 0; j < BATCH; ++j) {
        const int k = k0 + j;
        const int p = reverse ? n - 1 - k : k;
        // first slot of each segment met in scan order: p*sub (prefix) or p*sub+sub-1 (suffix)
        if (k < n && (reverse ? (p % sub == sub - 1) : (p % sub == 0))) s[(size_t)p * E4] = acc;
        acc.x += v[j].x; acc.y += v[j].y; acc.z += v[j].z; acc.w += v[j].w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < BATCH; ++j) { acc.x += v[j].x; acc.y += v[j].y; acc.z += v[j].z; acc.w += v[j].w; }
    }
  }
  if (!causal) s[0] = acc;
}

// ---------------------------------------------------------------------------
// Sweep: carry-in state, then per chunk the readout (and, causal, the
// intra-chunk term and the state update).  Writes O and den.
// ---------------------------------------------------------------------------
// ADD: add this frequency group's numerator and denominator to the sums the
// earlier groups stored; the old sums are loaded at the start of each chunk,
// so their latency overlaps the chunk's work.
// CH: tokens per chunk of the causal sweep (16, 32 or 64; the intra-chunk
// term covers j <= i within a chunk, earlier tokens enter through the carried
// state).  Token contractions run in 32-token MFMA k-steps; a 16-token chunk
// pads its k-step with zero rows (staged once, never written).
template <class T, int D, int FW, int NW, bool NS, bool CAUSAL, int QG, bool ADD, int CH, bool MASK = false>
__global__ __launch_bounds__(NW * WAVE) void k_fwd_sweep(FwdArgs a) {
  typedef Shape<T, D, FW, NW, NS, CH> SH;
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, SH::NT, CH> StX;
  typedef RowStage<IO, SH::DV, SH::NT, CH> StV;
  constexpr int TT = CH / 16;                  // token tiles per chunk
  constexpr int KT = (CH + 31) / 32;           // 32-token k-steps per chunk
  constexpr int ROWS = KT * 32;                // token rows of the k-step operands
  static_assert(CH == 16 || CH == 32 || CH == 64, "chunk of 16, 32 or 64 tokens");
  static_assert(CAUSAL || CH == CHUNK, "the non-causal sweep uses 64-token chunks");
  constexpr int XV_N = CAUSAL ? ROWS * StV::LD : 8;
  constexpr int LDP = SH::FC * 16 + 4;     // [token][feature] rows of a wave's phi(K) block
  constexpr int PT_N = CAUSAL ? ROWS * LDP : 8;
  constexpr int C4 = SH::DV / 4;                                // float4 columns of a row
  constexpr int NIT = (QG * 16 * C4 + SH::NT - 1) / SH::NT;    // readout items per thread and round
  static_assert(TT % QG == 0, "whole reduction rounds per chunk");
  __shared__ __attribute__((aligned(16))) IO XQ[StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XK[CAUSAL ? StX::LDS_ELEMS : 8];
  __shared__ typename StX::Ssq SSQ[CH], SSK[CH];
  __shared__ __attribute__((aligned(16))) IO XV[XV_N];   // [token][value col]
  __shared__ __attribute__((aligned(16))) T PT[NW][PT_N];
  __shared__ __attribute__((aligned(16))) float RED[NW][QG * 16][SH::RPAD];

  // causal: one workgroup per segment; non-causal: per group of chunks (every
  // chunk reads the same total state)
  const WgCoord wc = wg_coord(a.sweep_groups, a.H, a.BH);
  const int seg = wc.seg, bh = wc.bh, h = bh % a.H;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const int fv = slice_valid<MASK, FW>(a.fvalid, w);
  const int nch = (a.N + CH - 1) / CH;
  const int c0 = seg * a.sweep_cps;
  const int c1 = min(c0 + a.sweep_cps, nch);
  const IO* Q = static_cast<const IO*>(a.Q) + (size_t)bh * a.N * D;
  const IO* K = static_cast<const IO*>(a.K) + (size_t)bh * a.N * D;
  const IO* V = static_cast<const IO*>(a.V) + (size_t)bh * a.N * SH::DV;
  IO* O = static_cast<IO*>(a.O) + (size_t)bh * a.N * SH::DV;
  float* den = a.den ? a.den + (size_t)bh * a.N : nullptr;

  StX sq, sk;
  StV sv;
  if (c0 < c1) {
    sq.fetch(Q, c0 * CH, a.N);
    if (CAUSAL) sk.fetch(K, c0 * CH, a.N);
    if (CAUSAL) sv.fetch(V, c0 * CH, a.N);
  }
  if (CAUSAL && CH < ROWS) {
    // zero k-step padding rows of V and of this wave's phi(K) block (both
    // zero, so no product with uninitialised LDS enters a sum)
    for (int i = threadIdx.x; i < (ROWS - CH) * StV::LD; i += SH::NT) XV[CH * StV::LD + i] = IO(0);
    for (int i = l; i < (ROWS - CH) * LDP; i += WAVE) PT[w][CH * LDP + i] = T(0.0f);
  }
  const auto inv_c = inv_c_of<T>(a.tau[h]);

  // carry-in state (exclusive prefix for causal, total for non-causal)
  f32x4 S[SH::FC][SH::DVT1];
  {
    const float* blk = a.state + (size_t)bh * a.segments * a.sub * SH::STATE + (size_t)w * SH::WAVE_STATE;
    if (CAUSAL && a.fold) {
      // the exclusive prefix of the local states, summed in the scan's order
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
        for (int dt = 0; dt < SH::DVT1; ++dt) S[fc][dt] = zero4();
      for (int k = 0; k < seg * a.sub; ++k) {
        const float* in = blk + (size_t)k * SH::STATE;
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
          for (int dt = 0; dt < SH::DVT1; ++dt)
            S[fc][dt] += *reinterpret_cast<const f32x4*>(in + ((fc * SH::DVT1 + dt) * WAVE + l) * 4);
      }
    } else {
      const float* in = blk + (size_t)(CAUSAL ? seg * a.sub : 0) * SH::STATE;
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
        for (int dt = 0; dt < SH::DVT1; ++dt)
          S[fc][dt] = *reinterpret_cast<const f32x4*>(in + ((fc * SH::DVT1 + dt) * WAVE + l) * 4);
    }
  }
  const Frag<T> ones = ones_col0<T>();
  // projection fragments, held for the whole sweep: built from W by each wave
  FreqSlice<T, D, FW, NS> fs;
  fs.load(a.W1 + (size_t)h * a.w_stride, NS ? a.W2 + (size_t)h * a.w_stride : nullptr, w * FW);
  Frag<T> sf[SH::DVT1][SH::FT];
  if (!CAUSAL) {
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) sf[dt][ft] = pair_tiles<T>(S[2 * ft][dt], S[2 * ft + 1][dt]);
  }

  for (int c = c0; c < c1; ++c) {
    const int tok0 = c * CH;
    // no barrier before the staging stores: every read of the staging buffers
    // (projections, value fragments) precedes the previous chunk's last
    // readout barrier
    sq.store(XQ, SSQ);
    if (CAUSAL) sk.store(XK, SSK);
    if (CAUSAL) sv.store(XV);
    __syncthreads();
    // next chunk's rows
    {
      const int t1 = c + 1 < c1 ? tok0 + CH : tok0;   // the last chunk refetches itself (unused)
      sq.fetch(Q, t1, a.N);
      if (CAUSAL) sk.fetch(K, t1, a.N);
      if (CAUSAL) sv.fetch(V, t1, a.N);
    }
    // the earlier groups' sums for this chunk (rows past N read row N-1, unused)
    float4 old_n[ADD ? TT / QG : 1][ADD ? NIT : 1];
    float old_d[ADD ? TT / QG : 1][ADD ? NIT : 1];
    if (ADD) {
#pragma unroll
      for (int q = 0; q < TT / QG; ++q)
#pragma unroll
        for (int k = 0; k < NIT; ++k) {
          const int it = threadIdx.x + k * SH::NT;
          const size_t row = (size_t)bh * a.N + min(tok0 + q * QG * 16 + it / C4, a.N - 1);
          if (it < QG * 16 * C4) {
            old_n[q][k] = *reinterpret_cast<const float4*>(a.acc_num + row * SH::DV + 4 * (it % C4));
            old_d[q][k] = a.acc_den[row];
          }
        }
    }

    Frag<T> pq[SH::FT][TT];
    Frag<T> pk[CAUSAL ? SH::FT : 1][TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      ProjT<T> p[SH::PR];
      typename StX::Ssq ssq;
      project_tile_lds<T, D, FW, NS, StX::LD>(fs, XQ, SSQ, tt, p, ssq);
      float sc = row_scale(ssq, inv_c, a.s_const, tok0 + tt * 16 + r < a.N);
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) pq[ft][tt] = features<T, SH::FT, NS>(p, ft, sc, fv);
      if (CAUSAL) {
        project_tile_lds<T, D, FW, NS, StX::LD>(fs, XK, SSK, tt, p, ssq);
        sc = row_scale(ssq, inv_c, a.s_const, tok0 + tt * 16 + r < a.N);
#pragma unroll
        for (int ft = 0; ft < SH::FT; ++ft) {
          pk[ft][tt] = features<T, SH::FT, NS>(p, ft, sc, fv);
          store_frag_nm<T>(PT[w], LDP, tt * 16, (2 * ft) * 16, (2 * ft + 1) * 16, pk[ft][tt]);
        }
      }
    }

    // state operand for the readout: rows = value columns, k = this wave's
    // features (the non-causal total state is converted once, before the loop)
    if (CAUSAL) {
#pragma unroll
      for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
        for (int ft = 0; ft < SH::FT; ++ft) sf[dt][ft] = pair_tiles<T>(S[2 * ft][dt], S[2 * ft + 1][dt]);
    }

    // intra-chunk kernel matrix, transposed: rows = key tokens, cols = query tokens
    Frag<T> ap[CAUSAL ? KT : 1][TT];
    if (CAUSAL) {
#pragma unroll
      for (int tq = 0; tq < TT; ++tq) {
        f32x4 at[TT];
#pragma unroll
        for (int tk = 0; tk < TT; ++tk) {
          at[tk] = zero4();
          if (tk <= tq) {
#pragma unroll
            for (int ft = 0; ft < SH::FT; ++ft) mma(at[tk], pk[ft][tk], pq[ft][tq]);
            if (tk == tq) {
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (4 * g + i > r) at[tk][i] = 0.f;
            }
          }
        }
#pragma unroll
        for (int ks = 0; ks < KT; ++ks) ap[ks][tq] = pair_tiles<T>(at[2 * ks], 2 * ks + 1 < TT ? at[(2 * ks + 1) % TT] : zero4());
      }
    }

    Frag<T> vf[CAUSAL ? SH::DVT : 1][KT];
    if (CAUSAL) {
#pragma unroll
      for (int dt = 0; dt < SH::DVT; ++dt)
#pragma unroll
        for (int ks = 0; ks < KT; ++ks) vf[dt][ks] = lds_tr_frag<T>(reinterpret_cast<const T*>(XV), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16);
    }

    // readout partials, reduced across waves in groups of QG query tiles
#pragma unroll
    for (int q0 = 0; q0 < TT; q0 += QG) {
      if (q0 > 0) __syncthreads();
#pragma unroll
      for (int qq = 0; qq < QG; ++qq) {
        const int tq = q0 + qq;
#pragma unroll
        for (int dt = 0; dt < SH::DVT1; ++dt) {
          f32x4 acc = zero4();
          if (CAUSAL) {
#pragma unroll
            for (int ks = 0; ks < KT; ++ks)
              if (32 * ks <= 16 * tq + 15) mma(acc, dt < SH::DVT ? vf[dt][ks] : ones, ap[ks][tq]);
          }
#pragma unroll
          for (int ft = 0; ft < SH::FT; ++ft) mma(acc, sf[dt][ft], pq[ft][tq]);
          *reinterpret_cast<f32x4*>(&RED[w][qq * 16 + r][dt * 16 + 4 * g]) = acc;
        }
      }
      if (CAUSAL && q0 + QG >= TT) {
        // state update S' += phi(K)^T [V | 1] with this wave's transposed phi(K)
#pragma unroll
        for (int ks = 0; ks < KT; ++ks)
#pragma unroll
          for (int fc = 0; fc < SH::FC; ++fc) {
            const Frag<T> pkt = lds_tr_frag<T>(PT[w], LDP, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, fc * 16);
#pragma unroll
            for (int dt = 0; dt < SH::DVT; ++dt) mma(S[fc][dt], pkt, vf[dt][ks]);
            mma(S[fc][SH::DVT], pkt, ones);
          }
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < NIT; ++k) {
        const int it = threadIdx.x + k * SH::NT;
        if (it >= QG * 16 * C4) break;
        const int t = it / C4, c4 = it % C4;
        const int tok = tok0 + q0 * 16 + t;
        float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
        float dn = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
          const float4 v = *reinterpret_cast<const float4*>(&RED[ww][t][4 * c4]);
          num.x += v.x; num.y += v.y; num.z += v.z; num.w += v.w;
          dn += RED[ww][t][SH::DV];
        }
        if (tok < a.N) {
          if (ADD || a.acc) {
            // one frequency group's share of the numerator and denominator
            float4* an = reinterpret_cast<float4*>(a.acc_num + ((size_t)bh * a.N + tok) * SH::DV + 4 * c4);
            float* ad = a.acc_den + (size_t)bh * a.N + tok;
            if (ADD) {
              const float4 p = old_n[q0 / QG][k];
              num.x += p.x; num.y += p.y; num.z += p.z; num.w += p.w;
              dn += old_d[q0 / QG][k];
            }
            *an = num;
            if (c4 == 0) *ad = dn;
          } else {
            // one reciprocal per row (v_rcp_f32, 1 ulp); den = 0 gives inf/NaN as num/0 does
            const float inv = __builtin_amdgcn_rcpf(dn);
            IO* o = O + (size_t)tok * SH::DV + 4 * c4;
            o[0] = float_to_io<IO>(num.x * inv);
            o[1] = float_to_io<IO>(num.y * inv);
            o[2] = float_to_io<IO>(num.z * inv);
            o[3] = float_to_io<IO>(num.w * inv);
            if (den && c4 == 0) den[tok] = dn;
          }
        }
      }
    }
  }
  if (CAUSAL && a.state_out && seg == a.sweep_groups - 1) {
    // causal prefill: the last segment ends with the state of the whole
    // sequence (an empty trailing segment holds it as its carry-in).  Tile
    // (fc, dt) has rows = features 4g+i of feature tile fc (fc = 2ft: cos of
    // frequency tile ft, 2ft+1: its sin) and cols = value columns; the
    // normaliser tile holds z in column 0.
    const size_t F2 = 2 * (size_t)a.state_m;
    const int sdv = a.state_dv;   // value columns of the state layout, <= SH::DV
    float* so = a.state_out + (size_t)bh * F2 * (sdv + 1);
    float* zo = so + F2 * sdv;
#pragma unroll
    for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int fl = w * FW + (fc / 2) * 16 + 4 * g + i;   // row within the group
        if (fl >= a.fvalid) continue;   // a padding row of a padded group
        const int f = a.state_f0 + fl;
        const size_t row = (fc % 2) ? (size_t)a.state_m + f : (size_t)f;
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt)
          if (dt * 16 + r < sdv) so[row * sdv + dt * 16 + r] = S[fc][dt][i];
        if (r == 0) zo[row] = S[fc][SH::DVT][i];
      }
  }
}

// Four consecutive values of one row as one vector store in the io dtype.
template <class IO>
__device__ __forceinline__ void store4(IO* p, const float (&v)[4]);
template <>
__device__ __forceinline__ void store4<u16>(u16* p, const float (&v)[4]) {
  const uint2 w = make_uint2((uint32_t)float_to_bf16_bits(v[0]) | ((uint32_t)float_to_bf16_bits(v[1]) << 16),
                             (uint32_t)float_to_bf16_bits(v[2]) | ((uint32_t)float_to_bf16_bits(v[3]) << 16));
  *reinterpret_cast<uint2*>(p) = w;
}
template <>
__device__ __forceinline__ void store4<float>(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}

// ---------------------------------------------------------------------------
// Non-causal readout with the tokens split across waves (bf16, m_eff <= 64).
// Every chunk reads the same total state, so each of the four waves takes one
// 16-token tile of a 64-token chunk over all 2m features: the total state is
// held by every wave as bf16 operand fragments (rows = value columns, k = the
// 32 features of one frequency tile, [cos | sin] as the feature fragments),
// and each wave projects its tokens onto all m frequencies.  No partial sums
// cross waves, so the only barrier per chunk is the staging one.
// ---------------------------------------------------------------------------
template <class T, int D, int M, bool NS, bool MASK = false>
__global__ __launch_bounds__(4 * WAVE) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_fwd_readout(FwdArgs a) {
  constexpr int NWR = 4;                        // waves: one 16-token tile each
  constexpr int FT = M / 16;                    // frequency tiles (all of them)
  constexpr int DVT = D / 16, DVT1 = DVT + 1;
  typedef FreqSlice<T, D, M, NS> FS;
  typedef Shape<T, D, 16, M / 16, NS> SS;       // the state pre-pass's split: 16 frequencies per wave
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, NWR * WAVE> StX;
  static_assert(CHUNK == 16 * NWR, "one token tile per wave");
  __shared__ __attribute__((aligned(16))) IO XQ2[2][StX::LDS_ELEMS];
  __shared__ typename StX::Ssq SSQ2[2][CHUNK];

  const WgCoord wc = wg_coord(a.sweep_groups, a.H, a.BH);
  const int seg = wc.seg, bh = wc.bh, h = bh % a.H;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const int c0 = seg * a.sweep_cps;
  const int c1 = min(c0 + a.sweep_cps, a.nchunks);
  const IO* Q = static_cast<const IO*>(a.Q) + (size_t)bh * a.N * D;
  IO* O = static_cast<IO*>(a.O) + (size_t)bh * a.N * D;
  float* den = a.den ? a.den + (size_t)bh * a.N : nullptr;

  StX sq;
  if (c0 < c1) sq.fetch(Q, c0 * CHUNK, a.N);
  const auto inv_c = inv_c_of<T>(a.tau[h]);
  // total state (slot 0 of this slice after the scan): pre-pass wave ft holds
  // frequency tile ft, its tile fc = 0 the cos features and fc = 1 the sin ones
  Frag<T> sf[DVT1][FT];
  {
    const float* in = a.state + (size_t)bh * a.segments * a.sub * SS::STATE;
#pragma unroll
    for (int ft = 0; ft < FT; ++ft)
#pragma unroll
      for (int dt = 0; dt < DVT1; ++dt) {
        const float* blk = in + (size_t)ft * SS::WAVE_STATE;
        const f32x4 cs = *reinterpret_cast<const f32x4*>(blk + ((0 * DVT1 + dt) * WAVE + l) * 4);
        const f32x4 sn = *reinterpret_cast<const f32x4*>(blk + ((1 * DVT1 + dt) * WAVE + l) * 4);
        sf[dt][ft] = pair_tiles<T>(cs, sn);
      }
  }
  FS fs;
  fs.load(a.W1 + (size_t)h * a.w_stride, NS ? a.W2 + (size_t)h * a.w_stride : nullptr, 0);

  for (int c = c0; c < c1; ++c) {
    // double-buffered staging: the chunk that last read this buffer (two back)
    // is separated from this store by the previous chunk's barrier
    const int par = (c - c0) & 1;
    IO* XQ = XQ2[par];
    typename StX::Ssq* SSQ = SSQ2[par];
    const int tok0 = c * CHUNK;
    sq.store(XQ, SSQ);
    sq.fetch(Q, c + 1 < c1 ? tok0 + CHUNK : tok0, a.N);   // the last chunk refetches itself (unused)
    __syncthreads();
    ProjT<T> p[FS::PR];
    typename StX::Ssq ssq;
    project_tile_lds<T, D, M, NS, StX::LD>(fs, XQ, SSQ, w, p, ssq);
    const int tok = tok0 + w * 16 + r;
    const float sc = row_scale(ssq, inv_c, a.s_const, tok < a.N);
    f32x4 acc[DVT1];
#pragma unroll
    for (int dt = 0; dt < DVT1; ++dt) acc[dt] = zero4();
#pragma unroll
    for (int ft = 0; ft < FT; ++ft) {
      const Frag<T> pq = features<T, FT, NS>(p, ft, sc, MASK ? a.fvalid : M);
#pragma unroll
      for (int dt = 0; dt < DVT1; ++dt) mma(acc[dt], sf[dt][ft], pq);
    }
    // acc[dt]: rows = value columns dt*16 + 4g + i, column = token r; the
    // normaliser tile holds den in its row 0 (lane r of lane group 0)
    const float dn = __shfl(acc[DVT][0], r);
    const float inv = __builtin_amdgcn_rcpf(dn);   // den = 0 gives inf/NaN as num/0 does
    if (tok < a.N) {
#pragma unroll
      for (int dt = 0; dt < DVT; ++dt) {
        const float v[4] = {acc[dt][0] * inv, acc[dt][1] * inv, acc[dt][2] * inv, acc[dt][3] * inv};
        store4<IO>(O + (size_t)tok * D + dt * 16 + 4 * g, v);
      }
      if (den && g == 0) den[tok] = dn;
    }
  }
}

// ---------------------------------------------------------------------------
// Standalone feature map: Phi [B,H,N,2m], [cos | sin] blocks.  A workgroup
// walks a.chunks_per_seg consecutive chunks of one (b,h) slice with its
// frequency fragments built once; each lane writes its four consecutive
// features of a block as one vector store.
// ---------------------------------------------------------------------------
// The chunk's X rows are staged through LDS (prefetched a chunk ahead), every
// wave projects them for its frequency slice, and the features are gathered
// as [token][feature] rows in LDS, then written out as whole 16-byte vectors.
template <class T, int D, int FW, int NW, bool NS>
__global__ __launch_bounds__(NW * WAVE) void k_feature_map(FwdArgs a) {
  typedef Shape<T, D, FW, NW, NS> SH;
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, SH::NT> StX;
  constexpr int F = 2 * SH::M;                 // features per staged row
  constexpr int VEC = 16 / (int)sizeof(IO);    // elements per 16-byte vector
  constexpr int LDF = F + VEC;                 // row stride of the staged features
  __shared__ __attribute__((aligned(16))) IO XL[StX::LDS_ELEMS];
  __shared__ typename StX::Ssq SSQ[CHUNK];
  __shared__ __attribute__((aligned(16))) IO PH[CHUNK * LDF];
  const int bh = blockIdx.y, h = bh % a.H;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  // this launch covers frequencies [state_f0, state_f0 + fvalid) of state_m
  // (fvalid <= M, a multiple of 16): their cos and sin columns of rows of
  // 2 state_m features
  const int fv = a.fvalid, mo = a.state_m, f0o = a.state_f0;
  const int vrow = 2 * fv / VEC;               // output vectors per row
  const int nvo = CHUNK * vrow;
  const IO* X = static_cast<const IO*>(blockIdx.z ? a.K : a.Q) + (size_t)bh * a.N * D;
  IO* Phi = static_cast<IO*>(blockIdx.z ? a.O2 : a.O) + (size_t)bh * a.N * 2 * mo;
  const int c0 = blockIdx.x * a.chunks_per_seg;
  const int c1 = min(c0 + a.chunks_per_seg, a.nchunks);
  StX sx;
  if (c0 < c1) sx.fetch(X, c0 * CHUNK, a.N);
  FreqSlice<T, D, FW, NS> fs;   // frequencies past fvalid load as zero rows (their columns are not written)
  fs.template load<true>(a.W1 + (size_t)h * a.w_stride, NS ? a.W2 + (size_t)h * a.w_stride : nullptr, w * FW, fv);
  const auto inv_c = inv_c_of<T>(a.tau[h]);
  for (int c = c0; c < c1; ++c) {
    const int tok0 = c * CHUNK;
    __syncthreads();   // the previous chunk's reads of XL and PH are done
    sx.store(XL, SSQ);
    sx.fetch(X, c + 1 < c1 ? tok0 + CHUNK : tok0, a.N);   // the last chunk refetches itself (unused)
    __syncthreads();
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      ProjT<T> p[SH::PR];
      typename StX::Ssq ssq;
      project_tile_lds<T, D, FW, NS, StX::LD>(fs, XL, SSQ, tt, p, ssq);
      // the values are produced in fp32 and rounded once to the io dtype
      const float sc = row_scale(ssq, inv_c, a.s_const, tok0 + tt * 16 + r < a.N);
      IO* row = PH + (tt * 16 + r) * LDF;
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) {
        const Frag<float> f = features<float, SH::FT, NS>(p, ft, sc);
        const int f0 = w * FW + ft * 16 + 4 * g;
        const float cv[4] = {f.get(0), f.get(1), f.get(2), f.get(3)};
        const float sv[4] = {f.get(4), f.get(5), f.get(6), f.get(7)};
        store4<IO>(row + f0, cv);
        store4<IO>(row + SH::M + f0, sv);
      }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < nvo; v += SH::NT) {
      const int t = v / vrow, j = v % vrow;
      const int part = j / (fv / VEC), cv = j % (fv / VEC);   // cos block, then sin block
      if (tok0 + t < a.N)
        *reinterpret_cast<uint4*>(Phi + (size_t)(tok0 + t) * 2 * mo + part * mo + f0o + cv * VEC) =
            *reinterpret_cast<const uint4*>(PH + t * LDF + part * SH::M + cv * VEC);
    }
  }
}

// ---------------------------------------------------------------------------
// After the last frequency group: O = num / den from the fp32 sums, den out.
// One thread per 4 value columns of one row.
// ---------------------------------------------------------------------------
template <class IO>
__global__ __launch_bounds__(256) void k_fwd_finish(FwdArgs a, int dv) {
  const size_t rows = (size_t)a.BH * a.N;
  const int c4n = dv / 4;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * c4n) return;
  const size_t row = i / c4n;
  const int c4 = (int)(i % c4n);
  const float4 num = *reinterpret_cast<const float4*>(a.acc_num + row * dv + 4 * c4);
  const float dn = a.acc_den[row];
  const float inv = __builtin_amdgcn_rcpf(dn);
  IO* o = static_cast<IO*>(a.O) + row * dv + 4 * c4;
  o[0] = float_to_io<IO>(num.x * inv);
  o[1] = float_to_io<IO>(num.y * inv);
  o[2] = float_to_io<IO>(num.z * inv);
  o[3] = float_to_io<IO>(num.w * inv);
  if (a.den && c4 == 0) a.den[row] = dn;
}

// ---------------------------------------------------------------------------
// Frequency rows of a padded group: dst[h][rows][d] holds the group's
// rows_valid rows of W, then zero rows (their features are masked to zero).
// One thread per 4 elements.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_pad_rows(const float* src, float* dst, int rows_valid, int rows, int d,
                                                  int src_stride) {
  const int h = blockIdx.y;
  const int i4 = blockIdx.x * 256 + threadIdx.x;
  if (4 * i4 >= rows * d) return;
  const int row = 4 * i4 / d;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (row < rows_valid) v = *reinterpret_cast<const float4*>(src + (size_t)h * src_stride + 4 * i4);
  *reinterpret_cast<float4*>(dst + ((size_t)h * rows) * d + 4 * i4) = v;
}

hipError_t launch_pad_rows(const float* src, float* dst, int H, int rows_valid, int rows, int d, int src_stride,
                           hipStream_t st) {
  if (d % 4 != 0) return hipErrorInvalidValue;
  k_pad_rows<<<dim3((rows * d / 4 + 255) / 256, H), 256, 0, st>>>(src, dst, rows_valid, rows, d, src_stride);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Column padding and cropping between row-major matrices of two widths, in
// 16-byte units: dst[r][u] = src[r][u] for u < us, zero for us <= u < ud.
// One thread per 16-byte unit of dst.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_copy_cols(const uint4* src, int us, uint4* dst, int ud, size_t rows) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * (size_t)ud) return;
  const size_t r = i / (size_t)ud;
  const int u = (int)(i - r * (size_t)ud);
  dst[i] = u < us ? src[r * (size_t)us + u] : make_uint4(0u, 0u, 0u, 0u);
}

hipError_t launch_copy_cols(const void* src, int cols_src, void* dst, int cols_dst, size_t rows, int elem_bytes,
                            hipStream_t st) {
  if (elem_bytes <= 0 || (cols_src * elem_bytes) % 16 != 0 || (cols_dst * elem_bytes) % 16 != 0)
    return hipErrorInvalidValue;
  const int us = cols_src * elem_bytes / 16, ud = cols_dst * elem_bytes / 16;
  const size_t n = rows * (size_t)ud;
  if (n == 0) return hipSuccess;
  const size_t blocks = (n + 255) / 256;
  if (blocks > 0x7fffffffULL) return hipErrorInvalidValue;
  // a crop reads us units of each source row and copies only the first ud of them
  k_copy_cols<<<dim3((unsigned)blocks), 256, 0, st>>>(static_cast<const uint4*>(src), us,
                                                      static_cast<uint4*>(dst), ud, rows);
  return hipGetLastError();
}

hipError_t launch_fwd_finish(const FwdArgs& a, bool bf16, int dv, hipStream_t st) {
  const size_t n = (size_t)a.BH * a.N * (dv / 4);
  const dim3 grid((unsigned)((n + 255) / 256));
  if (bf16)
    k_fwd_finish<u16><<<grid, 256, 0, st>>>(a, dv);
  else
    k_fwd_finish<float><<<grid, 256, 0, st>>>(a, dv);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Host-side dispatch.
// ---------------------------------------------------------------------------
// Causal sweep launch for one chunk length CH (token tiles per cross-wave
// reduction round: fewer rounds where LDS allows).
template <class T, int D, int FW, int NW, bool NS, bool ADD, int CH, bool MASK>
static void launch_causal_sweep(const FwdArgs& a, dim3 grid, hipStream_t st) {
  typedef Shape<T, D, FW, NW, NS, CH> SH;
  constexpr int TTc = CH / 16;
  constexpr int QG0 = (SH::DV >= 128) ? 1 : (NW >= 8 ? 2 : TTc);
  constexpr int QG = QG0 < TTc ? QG0 : TTc;
  k_fwd_sweep<T, D, FW, NW, NS, true, QG, ADD, CH, MASK><<<grid, SH::NT, 0, st>>>(a);
}

// The token-split readout serves bf16 shapes whose projection onto all m
// frequencies fits one wave's registers (m_eff <= 64, state split 4 x 16).
template <class T, int D, int FW, int NW, bool NS>
struct ReadoutSplit {
  static constexpr bool value = IsBf16<T>::value && !NS && FW * NW == 64 && FW == 16 && D <= 64;
};

template <class T, int D, int FW, int NW, bool NS, bool ADD, bool MASK>
static void launch_sweep(const FwdArgs& a, bool causal, dim3 grid, hipStream_t st) {
  typedef Shape<T, D, FW, NW, NS> SH;
  if constexpr (!ADD && ReadoutSplit<T, D, FW, NW, NS>::value) {
    if (!causal && a.acc == 0) {   // it writes O itself, not a group's sums
      k_fwd_readout<T, D, FW * NW, NS, MASK><<<grid, 4 * WAVE, 0, st>>>(a);
      return;
    }
  }
  if (!causal) {
    // one token tile per round: the non-causal sweep then fits several workgroups per CU
    k_fwd_sweep<T, D, FW, NW, NS, false, 1, ADD, CHUNK, MASK><<<grid, SH::NT, 0, st>>>(a);
  } else if (a.sweep_chunk == 16) {
    launch_causal_sweep<T, D, FW, NW, NS, ADD, 16, MASK>(a, grid, st);
  } else if (a.sweep_chunk == 32) {
    launch_causal_sweep<T, D, FW, NW, NS, ADD, 32, MASK>(a, grid, st);
  } else {
    launch_causal_sweep<T, D, FW, NW, NS, ADD, 64, MASK>(a, grid, st);
  }
}

template <class T, int D, int FW, int NW, bool NS>
static hipError_t run_fwd_t(const FwdArgs& a, bool causal, hipStream_t st) {
  typedef Shape<T, D, FW, NW, NS> SH;
  const dim3 grid(a.sweep_groups * a.BH);
  const dim3 pgrid(a.pre_segs * a.sub * a.BH);
  // prepared fragments serve the state pre-pass at d > 64, which reloads them
  // per chunk; the other forward kernels build theirs from W once
  if (D > 64) k_prep_freqs<T, D, FW, NW, NS><<<dim3(a.H, NW, 1), WAVE, 0, st>>>(a.W1, a.W2, a.wfrag, a.w_stride);
  timing_mark(KC_FWD_STATE, st, true);
  // a padded frequency group (only the 64-frequency shape has one, and it
  // runs first, so it never adds) takes the masking kernel variants
  const bool masked = a.fvalid < FW * NW;
  constexpr bool CAN_MASK = FW * NW == 64;
  if (masked && (!CAN_MASK || a.acc == 2)) return hipErrorInvalidValue;
  if (pgrid.x > 0) {
    if constexpr (CAN_MASK) {
      if (masked) k_fwd_state<T, D, FW, NW, NS, true><<<pgrid, SH::NT, 0, st>>>(a);
      else k_fwd_state<T, D, FW, NW, NS, false><<<pgrid, SH::NT, 0, st>>>(a);
    } else {
      k_fwd_state<T, D, FW, NW, NS, false><<<pgrid, SH::NT, 0, st>>>(a);
    }
  }
  timing_mark(KC_FWD_STATE, st, false);
  if (!a.fold) {
    const hipError_t e =
        launch_state_scan(a.state, nullptr, a.BH, a.segments, a.sub, SH::STATE, causal, st, a.pre_segs * a.sub);
    if (e != hipSuccess) return e;
  }
  timing_mark(KC_FWD_SWEEP, st, true);
  // At d = 64, m = 128 the sweep runs 4 waves of 32 frequencies (one wave per
  // SIMD; the readout's cross-wave reduction then covers a whole 64-token
  // chunk in one round), the state pre-pass 8 waves of 16.  Both keep the
  // states in the same layout: feature tile 2f + (0: cos, 1: sin) of
  // frequency tile f, whatever wave holds it.
  constexpr int FWS = (D == 64 && FW * NW == 128) ? 32 : FW;
  constexpr int NWS = FW * NW / FWS;
  // a later frequency group adds to the earlier groups' sums
  if (a.acc == 2) {
    launch_sweep<T, D, FWS, NWS, NS, true, false>(a, causal, grid, st);
  } else if (masked) {
    if constexpr (CAN_MASK) launch_sweep<T, D, FWS, NWS, NS, false, true>(a, causal, grid, st);
  } else {
    launch_sweep<T, D, FWS, NWS, NS, false, false>(a, causal, grid, st);
  }
  timing_mark(KC_FWD_SWEEP, st, false);
  return hipGetLastError();
}

template <class T, int D, int FW, int NW, bool NS>
static hipError_t run_fmap_t(const FwdArgs& a, hipStream_t st) {
  typedef Shape<T, D, FW, NW, NS> SH;
  dim3 grid((a.nchunks + a.chunks_per_seg - 1) / a.chunks_per_seg, a.BH, a.K ? 2 : 1);
  timing_mark(KC_FEATURE_MAP, st, true);
  k_feature_map<T, D, FW, NW, NS><<<grid, SH::NT, 0, st>>>(a);
  timing_mark(KC_FEATURE_MAP, st, false);
  return hipGetLastError();
}

template <class T, int D, int FW, int NW>
static hipError_t run_attn_v(const FwdArgs& a, bool ns, bool causal, hipStream_t st) {
  return ns ? run_fwd_t<T, D, FW, NW, true>(a, causal, st) : run_fwd_t<T, D, FW, NW, false>(a, causal, st);
}
template <class T, int D, int FW, int NW>
static hipError_t run_fmap_v(const FwdArgs& a, bool ns, hipStream_t st) {
  return ns ? run_fmap_t<T, D, FW, NW, true>(a, st) : run_fmap_t<T, D, FW, NW, false>(a, st);
}

// Feature map shapes (d, m) and attention shapes (d, m of one frequency group).
hipError_t launch_fwd(const FwdArgs& a, const KernelShape& ks, bool fmap, hipStream_t st) {
  const bool ns = ks.nonstationary, causal = ks.causal;
  if (fmap) {
    if (ks.bf16) {
      if (ks.d == 32 && ks.m == 64) return run_fmap_v<__bf16, 32, 16, 4>(a, ns, st);
      if (ks.d == 64 && ks.m == 64) return run_fmap_v<__bf16, 64, 16, 4>(a, ns, st);
      if (ks.d == 64 && ks.m == 128) return run_fmap_v<__bf16, 64, 16, 8>(a, ns, st);
      if (ks.d == 128 && ks.m == 256) return run_fmap_v<__bf16, 128, 32, 8>(a, ns, st);
    } else {
      if (ks.d == 32 && ks.m == 64) return run_fmap_v<float, 32, 16, 4>(a, ns, st);
    }
    return hipErrorInvalidValue;
  }
  if (ks.bf16) {
    if (ks.d == 32 && ks.m == 64) return run_attn_v<__bf16, 32, 16, 4>(a, ns, causal, st);
    if (ks.d == 64 && ks.m == 64) return run_attn_v<__bf16, 64, 16, 4>(a, ns, causal, st);
    if (ks.d == 64 && ks.m == 128) return run_attn_v<__bf16, 64, 16, 8>(a, ns, causal, st);
    if (ks.d == 128 && ks.m == 64) return run_attn_v<__bf16, 128, 16, 4>(a, ns, causal, st);
  } else {
    if (ks.d == 32 && ks.m == 64) return run_attn_v<float, 32, 16, 4>(a, ns, causal, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_state_scan(float* state, float* state_rev, int BH, int P, int sub, int E, bool causal,
                             hipStream_t st, int nread) {
  if (E % 4 != 0) return hipErrorInvalidValue;   // the scan moves 4 floats per thread
  dim3 sgrid((E / 4 + 255) / 256, BH, (state && state_rev) ? 2 : 1);
  timing_mark(KC_SCAN, st, true);
  if (state)
    k_state_scan<<<sgrid, 256, 0, st>>>(state, state_rev, P, sub, E, causal ? 1 : 0, 0, nread);
  else
    k_state_scan<<<sgrid, 256, 0, st>>>(state_rev, nullptr, P, sub, E, causal ? 1 : 0, 1, P * sub);
  timing_mark(KC_SCAN, st, false);
  return hipGetLastError();
}

template <class T, int D, int FW, bool NS>
static size_t wfrag_bytes_t(int H, int NW) {
  return (size_t)H * NW * FragBlock<T, D, FW, NS>::PER_WAVE * sizeof(Frag<T>);
}

size_t wfrag_bytes(const KernelShape& ks, int H) {
  const bool ns = ks.nonstationary;
  if (ks.bf16) {
    if (ks.d == 32 && ks.m == 64) return ns ? wfrag_bytes_t<__bf16, 32, 16, true>(H, 4) : wfrag_bytes_t<__bf16, 32, 16, false>(H, 4);
    if (ks.d == 64 && ks.m == 64) return ns ? wfrag_bytes_t<__bf16, 64, 16, true>(H, 4) : wfrag_bytes_t<__bf16, 64, 16, false>(H, 4);
    if (ks.d == 64 && ks.m == 128) return ns ? wfrag_bytes_t<__bf16, 64, 16, true>(H, 8) : wfrag_bytes_t<__bf16, 64, 16, false>(H, 8);
    if (ks.d == 128 && ks.m == 64) return ns ? wfrag_bytes_t<__bf16, 128, 16, true>(H, 4) : wfrag_bytes_t<__bf16, 128, 16, false>(H, 4);
  } else {
    if (ks.d == 32 && ks.m == 64) return ns ? wfrag_bytes_t<float, 32, 16, true>(H, 4) : wfrag_bytes_t<float, 32, 16, false>(H, 4);
  }
  return 0;
}

// Waves per workgroup of the forward attention kernels of a shape.
int fwd_state_waves(const KernelShape& ks) { return (ks.bf16 && ks.d == 64 && ks.m == 128) ? 8 : 4; }

// Workgroups of the forward state pre-pass that run on one CU at a time, from
// the waves per SIMD its launch attributes fix.
int fwd_state_wgs_per_cu(const KernelShape& ks) {
  const int per_simd = state_waves_per_eu(ks.d, ks.nonstationary);
  const int wg_per_simd = fwd_state_waves(ks) / 4;
  return per_simd >= wg_per_simd ? per_simd / wg_per_simd : 1;
}

size_t fwd_state_floats(const KernelShape& ks) {
  const int fw = (ks.m == 64) ? 16 : 32;
  const int nw = ks.m / fw;
  const int fc = 2 * (fw / 16);
  return (size_t)nw * fc * (ks.d / 16 + 1) * WAVE * 4;
}

}  // namespace flex
