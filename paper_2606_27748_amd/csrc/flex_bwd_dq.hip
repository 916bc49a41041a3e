// dQ sweep of the RFF linear attention backward (the derivation and the
// kernel list are in flex_bwd.hip).  A translation unit of its own, so that
// it can be compiled with MFMA results placed in VGPRs, which suits this
// sweep (its results mostly feed vector code) but not the others.
#include "flex_bwd_common.hpp"

namespace flex {

// ---------------------------------------------------------------------------
// dQ: ascending sweep with the key-side prefix state S'.
// ---------------------------------------------------------------------------
// ACC: add dQ to the values an earlier frequency group stored (loaded at the
// start of each chunk, ahead of the next chunk's prefetch).
// WR: this sweep also does the pre-pass's query-side work (used when the
// forward's key-side states are passed in, so no pre-pass runs): the per-token
// 1/den and delta = dO . O, from the staging registers, written for the dK/dV
// sweep, and the segment-local R'^T = sum [dO | -delta]^T-rows x phi(Q)/den.
template <class T, int D, int FW, int NW, bool NS, bool CAUSAL, bool ACC, bool WR, bool MASK = false>
__global__ __launch_bounds__(NW * WAVE) void k_bwd_dq(BwdArgs a) {
  typedef Shape<T, D, FW, NW, NS, BWD_CHUNK> SH;
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, SH::NT, SH::CH> StX;
  typedef RowStage<IO, SH::DV, SH::NT, SH::CH> StV;
  typedef WTSlice<T, D, FW, NS> WTS;
  constexpr int DT = D / 16;
  constexpr int KG = (SH::DVT1 + 1) / 2;        // k-steps over [dO | -delta]
  constexpr int NOT = (DT * SH::TT + NW - 1) / NW;   // dQ tiles per wave (at most)
  // staging is double-buffered by chunk parity where LDS allows (d <= 64)
  constexpr int NBUF = D <= 64 ? 2 : 1;
  __shared__ __attribute__((aligned(16))) IO XQ2[NBUF][StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XK2[NBUF][StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XV2[NBUF][StV::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XDO2[NBUF][StV::LDS_ELEMS];
  constexpr int LDP = SH::FC * 16 + 4;          // row stride of the per-wave [token][row] blocks
  __shared__ __attribute__((aligned(16))) T PT[NW][SH::CH * LDP];   // dP, [token][projection row]
  __shared__ __attribute__((aligned(16))) float DWL[NW][SH::PR * DT * WAVE * 4];
  __shared__ float GS2[NBUF][SH::CH][2];
  __shared__ typename StX::Ssq SSQ2[NBUF][SH::CH];
  __shared__ __attribute__((aligned(16))) float SCK2[NBUF][SH::CH];   // per-token key scale s e(k)
  // dX fragments of every wave's projection rows, copied to LDS once per
  // workgroup: the dQ tiles read them there instead of from the L2 cache
  // every chunk
  constexpr int NDX = FragBlock<T, D, FW, NS>::NT_ * WAVE;   // fragments per wave
  constexpr bool DX_LDS = true;
  __shared__ Frag<T> DXL[DX_LDS ? NW : 1][DX_LDS ? NDX : 1];

  const WgCoord wc = wg_coord(a.segments, a.H, a.BH);
  const int seg = wc.seg, bh = wc.bh, h = bh % a.H;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const int fv = slice_valid<MASK, FW>(a.fvalid, w);
  const int c0 = seg * a.chunks_per_seg;
  const int c1 = min(c0 + a.chunks_per_seg, a.nchunks);
  const IO* Q = static_cast<const IO*>(a.Q) + (size_t)bh * a.N * D;
  const IO* K = static_cast<const IO*>(a.K) + (size_t)bh * a.N * D;
  const IO* V = static_cast<const IO*>(a.V) + (size_t)bh * a.N * SH::DV;
  const IO* dO = static_cast<const IO*>(a.dO) + (size_t)bh * a.N * SH::DV;
  float* gst = a.gstats + (size_t)bh * a.N * 2;
  float* dQ = a.dQ + (size_t)bh * a.N * D;
  // WR: thread v stages vectors v + i NT (i < PER) of Q, dO and O alike, so
  // the row sums dO . O come out of its staging registers
  static_assert(!WR || (StX::VPR == StV::VPR && StX::NV == StV::NV && (StV::NV <= SH::NT || StV::NV % SH::NT == 0)),
                "the same row vectors per thread for Q, dO and O");
  constexpr int WPER = WR ? StV::PER : 1;
  const IO* Ob = static_cast<const IO*>(a.O) + (size_t)bh * a.N * SH::DV;
  const float* den = a.den + (size_t)bh * a.N;
  float dn_next[WPER];
#pragma unroll
  for (int i = 0; i < WPER; ++i) dn_next[i] = 0.f;
  auto den_rows = [&](int t0) {   // rows past N (and threads past the rows) unused
#pragma unroll
    for (int i = 0; i < WPER; ++i)
      dn_next[i] = den[min(t0 + (int)(threadIdx.x + i * SH::NT) / StV::VPR, a.N - 1)];
  };

  StX sq, sk;
  StV sv, sdo, so;
  float2 gs_next = make_float2(0.f, 0.f);
  bool gs_ok = false;
  if (c0 < c1) {
    sq.fetch(Q, c0 * SH::CH, a.N); sk.fetch(K, c0 * SH::CH, a.N);
    sv.fetch(V, c0 * SH::CH, a.N); sdo.fetch(dO, c0 * SH::CH, a.N);
    if (WR) {
      so.fetch(Ob, c0 * SH::CH, a.N);
      den_rows(c0 * SH::CH);
    } else {
      gs_next = load_gs(gst, c0 * SH::CH, a.N, SH::CH, gs_ok);
    }
  }
  const Frag<T>* wproj = FragBlock<T, D, FW, NS>::proj(a.wfrag, h, NW, w);
  const Frag<T>* wdx = FragBlock<T, D, FW, NS>::dx(a.wfrag, h, NW, w);
  const auto inv_c = inv_c_of<T>(a.tau[h]);

  f32x4 ST[SH::DVT1][SH::FC];
  if (a.fstate && CAUSAL && a.ffold) {
    // the forward ran no scan: the exclusive prefix of its local states, summed
    // in the scan's order (the same sum the forward sweep formed)
    const float* blk = a.fstate + (size_t)bh * a.segments * a.fsub * SH::STATE;
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) ST[dt][fc] = zero4();
    for (int k = 0; k < seg * a.fsub; ++k) {
      const float* in = blk + (size_t)k * SH::STATE;
#pragma unroll
      for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc) ST[dt][fc] += fwd_state_tile_t<SH>(in, w, dt, fc);
    }
  } else if (a.fstate) {
    const float* in = a.fstate + ((size_t)bh * a.segments * a.fsub + (CAUSAL ? seg * a.fsub : 0)) * SH::STATE;
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) ST[dt][fc] = fwd_state_tile_t<SH>(in, w, dt, fc);
  } else {
    const float* in = a.sstate + ((size_t)bh * a.segments + (CAUSAL ? seg : 0)) * SH::STATE;
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc)
        ST[dt][fc] = *reinterpret_cast<const f32x4*>(in + state_off<SH>(w, dt, fc, l));
  }
  for (int i = l; i < SH::PR * DT * WAVE; i += WAVE)
    *reinterpret_cast<f32x4*>(&DWL[w][i * 4]) = zero4();
  if constexpr (DX_LDS) {   // ordered before the first dQ tile by the first staging barrier
    for (int i = threadIdx.x; i < NW * NDX; i += SH::NT)
      DXL[i / NDX][i % NDX] = FragBlock<T, D, FW, NS>::dx(a.wfrag, h, NW, i / NDX)[i % NDX];
  }
  const Frag<T> ones = ones_col01<T>();
  f32x4 RT[WR ? SH::DVT1 : 1][WR ? SH::FC : 1];
#pragma unroll
  for (int dt = 0; dt < (WR ? SH::DVT1 : 1); ++dt)
#pragma unroll
    for (int fc = 0; fc < (WR ? SH::FC : 1); ++fc) RT[dt][fc] = zero4();

  // projection fragments: held for the whole sweep at d <= 64 (without the
  // query-side states, which take those registers), else reloaded per chunk
  // ahead of the staging barriers
  constexpr bool KEEP_FS = D <= 64 && !WR;
  FreqSlice<T, D, FW, NS> fs;
  if (KEEP_FS) fs.load_frags(wproj);
  for (int c = c0; c < c1; ++c) {
    // This chunk's staging buffers.  Double-buffered, they need no barrier
    // before they are written: the chunk that last read them (two back) is
    // separated from this point by the previous chunk's barriers.
    const int par = NBUF == 2 ? (c - c0) & 1 : 0;
    IO* XQ = XQ2[par];
    IO* XK = XK2[par];
    IO* XV = XV2[par];
    IO* XDO = XDO2[par];
    float (*GS)[2] = GS2[par];
    typename StX::Ssq* SSQ = SSQ2[par];
    float* SCK = SCK2[par];
    const int tok0 = c * SH::CH;
    if (!KEEP_FS) fs.load_frags(wproj);
    // an earlier group's dQ of this chunk (rows past N read row N-1, unused)
    f32x4 old_q[ACC ? NOT : 1];
    if (ACC) {
#pragma unroll
      for (int k = 0; k < NOT; ++k) {
        const int ot = w + k * NW, dt = ot % DT, tt = ot / DT;
        const int tok = min(tok0 + tt * 16 + r, a.N - 1);
        if (ot < DT * SH::TT) old_q[k] = *reinterpret_cast<const f32x4*>(dQ + (size_t)tok * D + dt * 16 + 4 * g);
      }
    }
    if (NBUF == 1) __syncthreads();   // single buffer: the previous chunk's reads are done
    sq.store(XQ, SSQ);
    sk.store(XK, SCK, [&](int t, auto ssq) { return row_scale(ssq, inv_c, a.s_const, tok0 + t < a.N); });
    sv.store(XV); sdo.store(XDO);
    if constexpr (WR) {
      // 1/den and delta of this thread's rows (rows past N: zero vectors, delta 0)
#pragma unroll
      for (int i = 0; i < WPER; ++i) {
        const int v = threadIdx.x + i * SH::NT, t = v / StV::VPR;
        const bool mine = v < StV::NV;
        const bool ok = mine && tok0 + t < a.N;
        float dsum = 0.f;
        const uint4 x = sdo.vec(i), y = so.vec(i);
        const IO* ex = reinterpret_cast<const IO*>(&x);
        const IO* ey = reinterpret_cast<const IO*>(&y);
#pragma unroll
        for (int j = 0; j < StV::VEC; ++j) dsum += io_to_float(ex[j]) * io_to_float(ey[j]);
        dsum = lane_sum<StV::VPR>(dsum);
        if (mine && v % StV::VPR == 0) {
          const float inv = ok ? 1.0f / dn_next[i] : 0.f;
          GS[t][0] = inv;
          GS[t][1] = ok ? dsum : 0.f;
          if (ok) { gst[(size_t)(tok0 + t) * 2] = inv; gst[(size_t)(tok0 + t) * 2 + 1] = dsum; }
        }
      }
    } else {
      if (threadIdx.x < SH::CH) { GS[threadIdx.x][0] = gs_ok ? gs_next.x : 0.f; GS[threadIdx.x][1] = gs_ok ? gs_next.y : 0.f; }
    }
    {
      const int t1 = c + 1 < c1 ? tok0 + SH::CH : tok0;   // the last chunk refetches itself (unused)
      sq.fetch(Q, t1, a.N); sk.fetch(K, t1, a.N); sv.fetch(V, t1, a.N); sdo.fetch(dO, t1, a.N);
      if (WR) {
        so.fetch(Ob, t1, a.N);
        den_rows(t1);
      } else {
        gs_next = load_gs(gst, t1, a.N, SH::CH, gs_ok);
      }
    }
    __syncthreads();

    // phi(K) of this wave's features enters only contractions over the key
    // tokens: token-row fragments (k = tokens), no transpose
    Frag<T> pk[SH::KT][SH::FC];
#pragma unroll
    for (int ks = 0; ks < SH::KT; ++ks) feature_frags_rows<T, D, FW, NS, StX::LD>(fs, XK, SCK, ks, pk[ks], fv);
    // phi(Q)/den and its P2-derivative fragments (the 1/den of dphi(Q) is
    // carried by these: their products with dphi(Q) in the chain rule are the
    // same)
    Frag<T> phq[SH::FT][SH::TT], psq[SH::FT][SH::TT];
#pragma unroll
    for (int tt = 0; tt < SH::TT; ++tt) {
      ProjT<T> p[SH::PR];
      typename StX::Ssq ssq;
      project_tile_lds<T, D, FW, NS, StX::LD>(fs, XQ, SSQ, tt, p, ssq);
      const float sc = row_scale(ssq, inv_c, a.s_const, tok0 + tt * 16 + r < a.N) * GS[tt * 16 + r][0];
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) features_psi<T, SH::FT, NS>(p, ft, sc, phq[ft][tt], psq[ft][tt], fv);
    }
    if constexpr (WR) {
      // R'^T += [dO | -delta]^T-rows x phi(Q)/den, with phi(Q)/den as [token]
      // [feature] in this wave's LDS block (read transposed; the block takes
      // this wave's dP later, after these reads)
#pragma unroll
      for (int tt = 0; tt < SH::TT; ++tt)
#pragma unroll
        for (int ft = 0; ft < SH::FT; ++ft)
          store_frag_nm<T>(PT[w], LDP, tt * 16, (2 * ft) * 16, (2 * ft + 1) * 16, phq[ft][tt]);
#pragma unroll
      for (int ks = 0; ks < SH::KT; ++ks) {
        Frag<T> gt[SH::DVT1];
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt) gt[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XDO), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16);
        gt[SH::DVT] = delta_rows<T>(GS, ks);
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc) {
          const Frag<T> pq = lds_tr_frag<T>(PT[w], LDP, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, fc * 16);
#pragma unroll
          for (int dt = 0; dt < SH::DVT1; ++dt) mma(RT[dt][fc], gt[dt], pq);
        }
      }
    }
    // intra-chunk M^T[j][i] = dO_i . V_j - delta_i for j <= i (1/den_i applied later)
    Frag<T> mt[CAUSAL ? SH::KT : 1][SH::TT];
    if (CAUSAL) {
#pragma unroll
      for (int tq = 0; tq < SH::TT; ++tq) {
        const float dl = GS[tq * 16 + r][1];
        f32x4 m[SH::TT];
#pragma unroll
        for (int tk = 0; tk < SH::TT; ++tk) {
          m[tk] = zero4();
          if (tk <= tq) {
#pragma unroll
            for (int kd = 0; kd < SH::DV / 32; ++kd) {
              Frag<T> av, bo;
              lds_row8(av, XV + (tk * 16 + r) * StV::LD, kd * 32 + 8 * g);
              lds_row8(bo, XDO + (tq * 16 + r) * StV::LD, kd * 32 + 8 * g);
              mma(m[tk], av, bo);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const bool keep = tk < tq || 4 * g + i <= r;
              m[tk][i] = keep ? m[tk][i] - dl : 0.f;
            }
          }
        }
#pragma unroll
        for (int ks = 0; ks < SH::KT; ++ks) mt[ks][tq] = pair_tiles<T>(m[2 * ks], m[2 * ks + 1]);
      }
    }
    // den * dphi(Q)^T[feature][query] = phi(K)^T M^T + S'^T-rows x [dO | -delta]
    f32x4 dph[SH::FC][SH::TT];
#pragma unroll
    for (int tq = 0; tq < SH::TT; ++tq) {
      Frag<T> gf[KG];
#pragma unroll
      for (int kd = 0; kd < KG; ++kd) {
        if (32 * kd < SH::DV) {
          gf[kd] = lds_tok_frag<T>(reinterpret_cast<const T*>(XDO) + (tq * 16 + r) * StV::LD, kd);
        } else {
          Frag<T> f;
          f.zero();
          float hi, lo;
          neg_split<T>(GS[tq * 16 + r][1], hi, lo);
          if (g == 0) { f.set(0, hi); f.set(1, lo); }
          gf[kd] = f;
        }
      }
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) {
        f32x4 acc = zero4();
        if (CAUSAL) {
#pragma unroll
          for (int ks = 0; ks < SH::KT; ++ks)
            if (32 * ks <= 16 * tq + 15) mma(acc, pk[ks][fc], mt[ks][tq]);
        }
#pragma unroll
        for (int kd = 0; kd < KG; ++kd) {
          const f32x4 z = zero4();
          const Frag<T> sp = pair_tiles<T>(ST[2 * kd][fc], 2 * kd + 1 < SH::DVT1 ? ST[2 * kd + 1][fc] : z);
          mma(acc, sp, gf[kd]);
        }
        dph[fc][tq] = acc;
      }
    }
    if (CAUSAL) {
      // S'^T += [V | 1]^T-rows x phi(K)
#pragma unroll
      for (int ks = 0; ks < SH::KT; ++ks) {
        Frag<T> vt[SH::DVT];
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt) vt[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XV), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16);
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc) {
#pragma unroll
          for (int dt = 0; dt < SH::DVT; ++dt) mma(ST[dt][fc], vt[dt], pk[ks][fc]);
          mma(ST[SH::DVT][fc], ones, pk[ks][fc]);
        }
      }
    }
    // chain rule through phi(Q): dP per radian, tiles [projection row tile][token tile]
    f32x4 dp[SH::PR][SH::TT];
#pragma unroll
    for (int tt = 0; tt < SH::TT; ++tt)
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) {
        f32x4 d2 = zero4();
        feature_grad<T, SH::FT, NS>(phq[ft][tt], psq[ft][tt], dph[2 * ft][tt], dph[2 * ft + 1][tt], dp[ft][tt], d2);
        if (NS) dp[SH::FT + ft][tt] = d2;
      }
    // dP of this wave as [token][projection row] in its LDS block
#pragma unroll
    for (int pr = 0; pr < SH::PR; ++pr)
#pragma unroll
      for (int tt = 0; tt < SH::TT; ++tt) store_tile_nm<T>(PT[w], LDP, tt * 16, pr * 16, dp[pr][tt]);
    __syncthreads();   // every wave's dP block complete
    // dQ = dP W' over all projection rows: each wave computes whole output
    // tiles dQ^T (d tile, token tile) from every wave's dP block and that
    // wave's dX fragments, so no cross-wave reduction is needed
    // (every tile's products first, then the stores: the dX fragment loads of
    // a later tile never wait behind an earlier tile's stores)
    f32x4 acc[NOT];
#pragma unroll
    for (int k = 0; k < NOT; ++k) {
      const int ot = w + k * NW;
      acc[k] = zero4();
      if (ot >= DT * SH::TT) continue;
      const int dt = ot % DT, tt = ot / DT;
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) {
        const Frag<T>* wd = DX_LDS ? DXL[ww] : FragBlock<T, D, FW, NS>::dx(a.wfrag, h, NW, ww);
#pragma unroll
        for (int ks = 0; ks < WTS::KP; ++ks) {
          Frag<T> b = load_frag_nm<T>(PT[ww], LDP, tt * 16, (2 * ks) * 16, (2 * ks + 1) * 16);
          if (2 * ks + 1 >= SH::PR) {   // no second row tile: keep unwritten LDS out of the product
#pragma unroll
            for (int j = 4; j < 8; ++j) b.set(j, 0.f);
          }
#pragma unroll
          for (int sp = 0; sp < WTS::NSPLIT; ++sp) mma(acc[k], wd[((sp * DT + dt) * WTS::KP + ks) * WAVE + l], b);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < NOT; ++k) {
      const int ot = w + k * NW;
      if (ot >= DT * SH::TT) continue;
      const int dt = ot % DT, tt = ot / DT;
      const int tok = tok0 + tt * 16 + r;
      if (tok < a.N) {
        if (ACC) acc[k] += old_q[k];   // later frequency groups add their share
        *reinterpret_cast<f32x4*>(dQ + (size_t)tok * D + dt * 16 + 4 * g) = acc[k];
      }
    }
    // frequency gradient partial: dW'[rows][d] += dP^T Q
    {
      // one 32-token k-step per chunk, added to the LDS partial one
      // projection-row tile at a time
      static_assert(SH::KT == 1, "one token k-step per chunk");
      Frag<T> xq[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) xq[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XQ), StX::LD, 4 * g, 16 + 4 * g, dt * 16);
#pragma unroll
      for (int pr = 0; pr < SH::PR; ++pr) {
        const Frag<T> dpt = lds_tr_frag<T>(PT[w], LDP, 4 * g, 16 + 4 * g, pr * 16);
        dw_mma_row<D, T>(DWL[w], pr, dpt, xq);
      }
    }
  }
  const size_t nmat = NS ? 2 : 1;
  float* out = a.dwpart + (((size_t)0 * a.BH + bh) * a.segments + seg) * nmat * SH::M * D;
#pragma unroll
  for (int pr = 0; pr < SH::PR; ++pr)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<f32x4*>(out + dw_tile_off<SH, D>(w, pr, dt, l)) =
          *reinterpret_cast<const f32x4*>(&DWL[w][((pr * DT + dt) * WAVE + l) * 4]);
  if constexpr (WR) {
    float* ro = a.rstate + ((size_t)bh * a.segments + seg) * SH::STATE;
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) *reinterpret_cast<f32x4*>(ro + state_off<SH>(w, dt, fc, l)) = RT[dt][fc];
  }
}

// Launch of the dQ sweep for one shape: grouped_acc adds into an earlier
// frequency group's dQ; wr does the pre-pass's query-side work
// (with the forward's key-side states).
template <class T, int D, int FW, int NW, bool NS, bool ACC, bool MASK>
static void launch_dq_acc(const BwdArgs& a, bool causal, bool wr, const dim3& grid, int nt, hipStream_t st) {
  if (wr) {
    if (causal) k_bwd_dq<T, D, FW, NW, NS, true, ACC, true, MASK><<<grid, nt, 0, st>>>(a);
    else k_bwd_dq<T, D, FW, NW, NS, false, ACC, true, MASK><<<grid, nt, 0, st>>>(a);
  } else {
    if (causal) k_bwd_dq<T, D, FW, NW, NS, true, ACC, false, MASK><<<grid, nt, 0, st>>>(a);
    else k_bwd_dq<T, D, FW, NW, NS, false, ACC, false, MASK><<<grid, nt, 0, st>>>(a);
  }
}

template <class T, int D, int FW, int NW, bool NS>
hipError_t launch_bwd_dq(const BwdArgs& a, bool causal, bool grouped_acc, bool wr, bool masked, hipStream_t st) {
  typedef Shape<T, D, FW, NW, NS, BWD_CHUNK> SA;
  const dim3 grid(a.segments * a.BH);
  if (masked) {   // a padded group: the 64-frequency shape, never adding
    if constexpr (FW * NW == 64) {
      if (!grouped_acc) {
        launch_dq_acc<T, D, FW, NW, NS, false, true>(a, causal, wr, grid, SA::NT, st);
        return hipGetLastError();
      }
    }
    return hipErrorInvalidValue;
  }
  if (grouped_acc)
    launch_dq_acc<T, D, FW, NW, NS, true, false>(a, causal, wr, grid, SA::NT, st);
  else
    launch_dq_acc<T, D, FW, NW, NS, false, false>(a, causal, wr, grid, SA::NT, st);
  return hipGetLastError();
}

#define FLEX_DQ_SHAPE(T, D, FW, NW)                                                                  \
  template hipError_t launch_bwd_dq<T, D, FW, NW, true>(const BwdArgs&, bool, bool, bool, bool, hipStream_t); \
  template hipError_t launch_bwd_dq<T, D, FW, NW, false>(const BwdArgs&, bool, bool, bool, bool, hipStream_t);
FLEX_DQ_SHAPE(__bf16, 32, 16, 4)
FLEX_DQ_SHAPE(__bf16, 64, 16, 4)
FLEX_DQ_SHAPE(__bf16, 64, 16, 8)
FLEX_DQ_SHAPE(__bf16, 128, 16, 4)
FLEX_DQ_SHAPE(float, 32, 16, 4)
#undef FLEX_DQ_SHAPE

}  // namespace flex
