// Backward kernels of the RFF linear attention (Eq.(linear att) with the
// Flexformer feature maps of Eq.(phi_n) / Eq.(phi_non)).  The paper gives no
// backward; this is the derivative of the forward:
//
//   [num|den]_i = sum_j a_ij [V_j ; 1],  a_ij = phi(Q_i).phi(K_j)  (j <= i if causal)
//   G_i = [dO_i ; -delta_i] / den_i,     delta_i = dO_i . O_i
//   dphi(Q_i) = S'_i G_i,   S'_i = sum_{j(<=i)} phi(K_j) [V_j;1]^T
//   dphi(K_j) = R'_j [V_j;1], R'_j = sum_{i(>=j)} phi(Q_i) G_i^T
//   dV_j = (R'_j^T phi(K_j))[:dv]
// then the feature-map chain rule (frequencies and norm factor exp(||x||^2/c)).
//
// Kernels (per (b,h) slice, sequence split into segments like the forward):
//   k_bwd_prepass : segment-local S'^T (key side) and R'^T (query side), and the
//                   per-token scalars 1/den_i, delta_i,
//   k_state_scan  : prefix of S' and suffix of R' over segments,
//   k_bwd_dq      : ascending chunk sweep carrying S'; dQ and the query-side
//                   frequency-gradient partials (flex_bwd_dq.hip),
//   k_bwd_dkv     : descending chunk sweep carrying R'; dK, dV, the key-side
//                   frequency-gradient partials and dtau partials,
//   k_bwd_reduce  : fixed-order sums of the partials into dW1, dW2, dtau.
// Waves split the frequencies as in the forward.  Both states are held as
// accumulator tiles with value columns as rows ([dv' x features]).
#include "flex_bwd_common.hpp"

namespace flex {

// ---------------------------------------------------------------------------
// Pre-pass: segment-local S'^T = sum [V;1]^T-rows x phi(K) and
// R'^T = sum [dO;-delta]^T-rows x phi(Q)/den; per-token 1/den and delta.
// ---------------------------------------------------------------------------
// WITH_S: also the key-side states S' (not needed when the forward's segment
// states are passed in).
// The pre-pass forms sums over a segment and per-token scalars only, so at
// d <= 64 it walks the segment in 64-token chunks (a backward segment is a
// whole number of them: it spans the forward's 64-token chunks), not the
// sweeps' 32; at d = 128 the double-buffered staging of 64 rows would not fit
// in LDS.
template <class T, int D, int FW, int NW, bool NS, bool WITH_S, bool MASK = false>
__global__ __launch_bounds__(NW * WAVE) void k_bwd_prepass(BwdArgs a) {
  // 64-token chunks where the staging fits: at d <= 64, and at d = 128 on the
  // query-side-only pass (K and V are not staged there)
  constexpr int PCH = (D <= 64 || !WITH_S) ? CHUNK : BWD_CHUNK;
  typedef Shape<T, D, FW, NW, NS, PCH> SH;
  static_assert(PCH % BWD_CHUNK == 0 && CHUNK % PCH == 0, "pre-pass chunks hold whole sweep chunks");
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, SH::NT, SH::CH> StX;
  typedef RowStage<IO, SH::DV, SH::NT, SH::CH> StV;
  // staging (and the per-token scalars) double-buffered by chunk parity
  __shared__ __attribute__((aligned(16))) IO XQ2[2][StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XK2[2][StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XDO2[2][StV::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XO2[2][StV::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XV2[2][StV::LDS_ELEMS];
  __shared__ float GS2[2][SH::CH][2];
  __shared__ float DEN2[2][SH::CH];
  __shared__ typename StX::Ssq SSQ2[2][SH::CH], SSK2[2][SH::CH];
  // per-token feature scales: s e(k) for keys, s e(q) / den for queries
  __shared__ __attribute__((aligned(16))) float SCK2[2][SH::CH], SCQ2[2][SH::CH];

  const WgCoord wc = wg_coord(a.segments, a.H, a.BH);
  const int seg = wc.seg, bh = wc.bh, h = bh % a.H;
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, r = l % 16, g = l / 16;
  const int fv = slice_valid<MASK, FW>(a.fvalid, w);
  const int cps = a.chunks_per_seg / (PCH / BWD_CHUNK);   // pre-pass chunks per segment
  const int c0 = seg * cps;
  const int c1 = min(c0 + cps, (a.N + SH::CH - 1) / SH::CH);
  const IO* Q = static_cast<const IO*>(a.Q) + (size_t)bh * a.N * D;
  const IO* K = static_cast<const IO*>(a.K) + (size_t)bh * a.N * D;
  const IO* V = static_cast<const IO*>(a.V) + (size_t)bh * a.N * SH::DV;
  const IO* dO = static_cast<const IO*>(a.dO) + (size_t)bh * a.N * SH::DV;
  const IO* Ob = static_cast<const IO*>(a.O) + (size_t)bh * a.N * SH::DV;
  const float* den = a.den + (size_t)bh * a.N;
  float* gst = a.gstats + (size_t)bh * a.N * 2;

  StX sq, sk;
  StV sv, sdo, so;
  // FUSED: every thread stages the same PER vectors of Q, dO and O (same
  // vectors per row, all threads busy), so the row sums dO . O and ||q||^2
  // come out of the staging registers with lane sums, and the per-token
  // scalars need no barrier of their own.  Each thread then loads den of its
  // own rows; otherwise thread t < CH loads that of row t.
  constexpr bool FUSED = StX::VPR == StV::VPR && StX::NV == StV::NV && StV::NV % SH::NT == 0;
  constexpr int FPER = FUSED ? StV::PER : 1;
  float dn_next[FPER];
#pragma unroll
  for (int i = 0; i < FPER; ++i) dn_next[i] = 0.f;
  auto den_rows = [&](int t0) {
#pragma unroll
    for (int i = 0; i < FPER; ++i) {
      const int t = FUSED ? (int)(threadIdx.x + i * SH::NT) / StV::VPR : (int)(threadIdx.x % SH::CH);
      dn_next[i] = den[min(t0 + t, a.N - 1)];   // rows past N unused
    }
  };
  if (c0 < c1) {
    sq.fetch(Q, c0 * SH::CH, a.N); sk.fetch(K, c0 * SH::CH, a.N);
    sv.fetch(V, c0 * SH::CH, a.N); sdo.fetch(dO, c0 * SH::CH, a.N); so.fetch(Ob, c0 * SH::CH, a.N);
    den_rows(c0 * SH::CH);
  }
  const Frag<T>* wproj = FragBlock<T, D, FW, NS>::proj(a.wfrag, h, NW, w);
  const auto inv_c = inv_c_of<T>(a.tau[h]);

  f32x4 ST[SH::DVT1][SH::FC], RT[SH::DVT1][SH::FC];
#pragma unroll
  for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
    for (int fc = 0; fc < SH::FC; ++fc) { ST[dt][fc] = zero4(); RT[dt][fc] = zero4(); }
  const Frag<T> ones = ones_col01<T>();
  constexpr int TPT = SH::NT / SH::CH;  // threads per token for the row reductions

  // projection fragments: held for the whole sweep on the query-side-only
  // pass at d <= 64, else reloaded per chunk ahead of the staging barriers
  constexpr bool KEEP_FS = D <= 64 && !WITH_S;
  FreqSlice<T, D, FW, NS> fs;
  if (KEEP_FS) fs.load_frags(wproj);
  for (int c = c0; c < c1; ++c) {
    // This chunk's buffers.  They need no barrier before they are written:
    // the chunk that last read them (two back) is separated from this point
    // by the previous chunk's barriers.
    const int par = (c - c0) & 1;
    IO* XQ = XQ2[par];
    IO* XK = XK2[par];
    IO* XDO = XDO2[par];
    IO* XO = XO2[par];
    IO* XV = XV2[par];
    float (*GS)[2] = GS2[par];
    float* DEN = DEN2[par];
    typename StX::Ssq* SSQ = SSQ2[par];
    typename StX::Ssq* SSK = SSK2[par];
    float* SCK = SCK2[par];
    float* SCQ = SCQ2[par];
    const int tok0 = c * SH::CH;
    if (!KEEP_FS) fs.load_frags(wproj);
    if constexpr (FUSED) {
      // per-token 1/den and delta = dO . O of this thread's rows (rows past N
      // are zero vectors: delta 0)
      float inv[FPER];
      bool ok[FPER];
#pragma unroll
      for (int i = 0; i < FPER; ++i) {
        const int t = (int)(threadIdx.x + i * SH::NT) / StV::VPR;
        ok[i] = tok0 + t < a.N;
        inv[i] = ok[i] ? 1.0f / dn_next[i] : 0.f;
        float dsum = 0.f;
        const uint4 x = sdo.vec(i), y = so.vec(i);
        const IO* ex = reinterpret_cast<const IO*>(&x);
        const IO* ey = reinterpret_cast<const IO*>(&y);
#pragma unroll
        for (int j = 0; j < StV::VEC; ++j) dsum += io_to_float(ex[j]) * io_to_float(ey[j]);
        dsum = lane_sum<StV::VPR>(dsum);
        if (threadIdx.x % StV::VPR == 0) {
          GS[t][0] = inv[i];
          GS[t][1] = ok[i] ? dsum : 0.f;
          if (ok[i]) { gst[(size_t)(tok0 + t) * 2] = inv[i]; gst[(size_t)(tok0 + t) * 2 + 1] = dsum; }
        }
      }
      sq.store_idx(XQ, SCQ, [&](int i, int, auto ssq) { return row_scale(ssq, inv_c, a.s_const, ok[i]) * inv[i]; });
      sdo.store(XDO);
    } else {
      sq.store(XQ, SSQ); sdo.store(XDO); so.store(XO);
      if (threadIdx.x < SH::CH) DEN[threadIdx.x] = dn_next[0];
    }
    if (WITH_S) {
      if constexpr (FUSED)
        sk.store(XK, SCK, [&](int t, auto ssq) { return row_scale(ssq, inv_c, a.s_const, tok0 + t < a.N); });
      else
        sk.store(XK, SSK);
      sv.store(XV);
    } else {   // K and V only warm the caches for the sweeps that follow
      sk.touch();
      sv.touch();
    }
    {
      const int t1 = c + 1 < c1 ? tok0 + SH::CH : tok0;   // the last chunk refetches itself (unused)
      sq.fetch(Q, t1, a.N); sk.fetch(K, t1, a.N);
      sv.fetch(V, t1, a.N); sdo.fetch(dO, t1, a.N); so.fetch(Ob, t1, a.N);
      den_rows(t1);
    }
    __syncthreads();
    // per-token 1/den and delta = dO . O (FUSED: done above)
    if constexpr (!FUSED) {
      const int t = threadIdx.x / TPT, part = threadIdx.x % TPT;
      float s = 0.f;
      for (int cidx = part; cidx < SH::DV; cidx += TPT)
        s += io_to_float(XDO[t * StV::LD + cidx]) * io_to_float(XO[t * StV::LD + cidx]);
      s = lane_sum<TPT>(s);
      if (part == 0) {
        const bool ok = tok0 + t < a.N;
        const float inv = ok ? 1.0f / DEN[t] : 0.f;
        GS[t][0] = inv;
        GS[t][1] = ok ? s : 0.f;
        if (WITH_S) SCK[t] = row_scale(SSK[t], inv_c, a.s_const, ok);
        SCQ[t] = row_scale(SSQ[t], inv_c, a.s_const, ok) * inv;
        if (ok) { gst[(size_t)(tok0 + t) * 2] = inv; gst[(size_t)(tok0 + t) * 2 + 1] = s; }
      }
      __syncthreads();
    }
    // both feature maps enter only the token sums: token-row features, no
    // transpose; the key side and the query side one after the other
#pragma unroll
    for (int ks = 0; ks < SH::KT; ++ks) {
      // value-side operands: rows = value columns, k = chunk tokens
      if constexpr (WITH_S) {
        Frag<T> vt[SH::DVT1], pk[SH::FC];
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt) vt[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XV), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16);
        vt[SH::DVT] = ones;
        feature_frags_rows<T, D, FW, NS, StX::LD>(fs, XK, SCK, ks, pk, fv);
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
          for (int dt = 0; dt < SH::DVT1; ++dt) mma(ST[dt][fc], vt[dt], pk[fc]);
      }
      {
        Frag<T> gt[SH::DVT1], pq[SH::FC];
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt) gt[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XDO), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16);
        gt[SH::DVT] = delta_rows<T>(GS, ks);
        feature_frags_rows<T, D, FW, NS, StX::LD>(fs, XQ, SCQ, ks, pq, fv);
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc)
#pragma unroll
          for (int dt = 0; dt < SH::DVT1; ++dt) mma(RT[dt][fc], gt[dt], pq[fc]);
      }
    }
  }
  float* so_ = a.sstate + ((size_t)bh * a.segments + seg) * SH::STATE;
  float* ro_ = a.rstate + ((size_t)bh * a.segments + seg) * SH::STATE;
#pragma unroll
  for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
    for (int fc = 0; fc < SH::FC; ++fc) {
      if (WITH_S) *reinterpret_cast<f32x4*>(so_ + state_off<SH>(w, dt, fc, l)) = ST[dt][fc];
      *reinterpret_cast<f32x4*>(ro_ + state_off<SH>(w, dt, fc, l)) = RT[dt][fc];
    }
}

// ---------------------------------------------------------------------------
// dK, dV: descending sweep with the query-side suffix state R'.
// ---------------------------------------------------------------------------
// ACC: add dK and dV to the values an earlier frequency group stored.  The
// old values are loaded at the start of each chunk, ahead of the next chunk's
// prefetch, so waiting for them never waits for that prefetch.
template <class T, int D, int FW, int NW, bool NS, bool CAUSAL, bool ACC, bool MASK = false>
__global__ __launch_bounds__(NW * WAVE) void k_bwd_dkv(BwdArgs a) {
  typedef Shape<T, D, FW, NW, NS, BWD_CHUNK> SH;
  typedef typename Io<T>::type IO;
  typedef RowStage<IO, D, SH::NT, SH::CH> StX;
  typedef RowStage<IO, SH::DV, SH::NT, SH::CH> StV;
  typedef WTSlice<T, D, FW, NS> WTS;
  constexpr int DT = D / 16;
  constexpr int KG = (SH::DVT1 + 1) / 2;
  constexpr int QG = (NW >= 8 || D >= 128) ? 1 : 2;
  constexpr int RP = SH::DV + 4;                 // row stride of the dV reduction rows
  constexpr int C4 = SH::DV / 4;                 // float4 columns of a dV row
  constexpr int NIT = (QG * 16 * C4 + SH::NT - 1) / SH::NT;   // dV items per thread and round
  constexpr int TT0STEP = DT < NW ? NW / DT : 1; // token-tile step of a wave's dK tiles
  constexpr int NDK = (DT + NW - 1) / NW;        // d tiles per wave (at most)
  constexpr int NTK = DT < NW ? (SH::TT + TT0STEP - 1) / TT0STEP : SH::TT;   // token tiles per d tile
  constexpr int RLP = SH::DV + 4;                // row stride of the bf16 R' copy, [feature][value col]
  constexpr int LDP = SH::FC * 16 + 4;           // row stride of the per-wave [token][row] blocks
  // Each wave owns one slot of REDRL: its bf16 copy of R' and, once its own
  // reads of that copy are done, its dV partials.  No other wave touches the
  // slot between the chunk's staging barrier and its dV reduction, so neither the
  // copy nor the partials need a barrier before they are written.
  constexpr int RED_W = QG * 16 * RP * 4;
  constexpr int RL_W = SH::FC * 16 * RLP * (int)sizeof(T);
  constexpr int SLOT = RED_W > RL_W ? RED_W : RL_W;
  // Staging is double-buffered by chunk parity where LDS allows (d <= 64).
  // There the next chunk is staged before this chunk's dP barrier, which then
  // also orders those stores before the next chunk's reads.  K rows and norms
  // are read after the dP barrier too (dK, dW', dtau), so they take three
  // buffers.
  constexpr int NBUF = D <= 64 ? 2 : 1;
  constexpr bool EARLY = NBUF == 2;
  constexpr int NKB = EARLY ? 3 : 1;
  __shared__ __attribute__((aligned(16))) IO XQ2[NBUF][StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XK2[NKB][StX::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XV2[NBUF][StV::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) IO XDO2[NBUF][StV::LDS_ELEMS];
  __shared__ __attribute__((aligned(16))) T PT[NW][SH::CH * LDP];   // phi(Q)/den, then dP: [token][row]
  __shared__ __attribute__((aligned(16))) char REDRL[NW * SLOT];
  __shared__ __attribute__((aligned(16))) float DWL[NW][SH::PR * DT * WAVE * 4];
  __shared__ float GS2[NBUF][SH::CH][2];
  __shared__ typename StX::Ssq SSQ2[NBUF][SH::CH], SSK2[NKB][SH::CH];
  __shared__ float TRED[SH::NT];
  __shared__ __attribute__((aligned(16))) float GP[SH::CH][NW][4];   // per-lane-group shares of g
  typedef float RedRow[QG * 16][RP];
  auto RED = [&](int ww) -> RedRow& { return *reinterpret_cast<RedRow*>(REDRL + ww * SLOT); };

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
  const float* gst = a.gstats + (size_t)bh * a.N * 2;
  float* dK = a.dK + (size_t)bh * a.N * D;
  T* RLw = reinterpret_cast<T*>(REDRL + w * SLOT);   // this wave's R' copy
  float* dV = a.dV + (size_t)bh * a.N * SH::DV;

  StX sq, sk;
  StV sv, sdo;
  float2 gs_next = make_float2(0.f, 0.f);
  bool gs_ok = false;
  if (c0 < c1) {
    const int t1 = (c1 - 1) * SH::CH;
    sq.fetch(Q, t1, a.N); sk.fetch(K, t1, a.N); sv.fetch(V, t1, a.N); sdo.fetch(dO, t1, a.N);
    gs_next = load_gs(gst, t1, a.N, SH::CH, gs_ok);
  }
  const Frag<T>* wproj = FragBlock<T, D, FW, NS>::proj(a.wfrag_kv, h, NW, w);
  const auto inv_c = inv_c_of<T>(a.tau[h]);

  f32x4 RT[SH::DVT1][SH::FC];
  if (CAUSAL && a.rfold) {
    // the suffix of the later segments' local states, summed in the scan's
    // order (last segment first)
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) RT[dt][fc] = zero4();
    for (int q = a.segments - 1; q > seg; --q) {
      const float* in = a.rstate + ((size_t)bh * a.segments + q) * SH::STATE;
#pragma unroll
      for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
        for (int fc = 0; fc < SH::FC; ++fc)
          RT[dt][fc] += *reinterpret_cast<const f32x4*>(in + state_off<SH>(w, dt, fc, l));
    }
  } else {
    const float* in = a.rstate + ((size_t)bh * a.segments + (CAUSAL ? seg : 0)) * SH::STATE;
#pragma unroll
    for (int dt = 0; dt < SH::DVT1; ++dt)
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc)
        RT[dt][fc] = *reinterpret_cast<const f32x4*>(in + state_off<SH>(w, dt, fc, l));
  }
  {
    // this wave's dW' partial starts from the query side's (dQ sweep) partial
    // of this workgroup position
    const size_t nmat = NS ? 2 : 1;
    const float* qpart = a.dwpart + (((size_t)0 * a.BH + bh) * a.segments + seg) * nmat * SH::M * D;
#pragma unroll
    for (int pr = 0; pr < SH::PR; ++pr)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<f32x4*>(&DWL[w][((pr * DT + dt) * WAVE + l) * 4]) =
            *reinterpret_cast<const f32x4*>(qpart + dw_tile_off<SH, D>(w, pr, dt, l));
  }
  float dtau_acc = 0.f;

  // dX fragments of this wave's d tile: held for the whole sweep when every
  // wave has one d tile (DT <= NW), else loaded per chunk ahead of the barrier
  Frag<T> wf[NW][WTS::KP][WTS::NSPLIT];
  auto load_wf = [&](int dt) {
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
      const Frag<T>* wd = FragBlock<T, D, FW, NS>::dx(a.wfrag_kv, h, NW, ww);
#pragma unroll
      for (int ks = 0; ks < WTS::KP; ++ks)
#pragma unroll
        for (int sp = 0; sp < WTS::NSPLIT; ++sp) wf[ww][ks][sp] = wd[((sp * DT + dt) * WTS::KP + ks) * WAVE + l];
    }
  };
  // held for the whole sweep with up to 4 waves; 8-wave workgroups (two
  // waves per SIMD, 256 registers) load them per chunk
  constexpr bool HOLD_WF = DT <= NW && NW <= 4;
  if (HOLD_WF) load_wf(w % DT);
  // Store the prefetched rows into the buffers of sweep step i and prefetch
  // chunk cn - 1 (chunk cn itself again when cn is the last one: the prefetch
  // is issued on every step, from an in-range chunk).
  auto stage = [&](int i, int cn) {
    const int par = NBUF == 2 ? i & 1 : 0, kp = i % NKB;
    sq.store(XQ2[par], SSQ2[par]); sk.store(XK2[kp], SSK2[kp]); sv.store(XV2[par]); sdo.store(XDO2[par]);
    if (threadIdx.x < SH::CH) {
      GS2[par][threadIdx.x][0] = gs_ok ? gs_next.x : 0.f;
      GS2[par][threadIdx.x][1] = gs_ok ? gs_next.y : 0.f;
    }
    const int t1 = (cn - 1 >= c0 ? cn - 1 : cn) * SH::CH;
    sq.fetch(Q, t1, a.N); sk.fetch(K, t1, a.N); sv.fetch(V, t1, a.N); sdo.fetch(dO, t1, a.N);
    gs_next = load_gs(gst, t1, a.N, SH::CH, gs_ok);
  };
  // Projection fragments, reloaded per chunk (held for the whole sweep they
  // would not fit the registers).
  FreqSlice<T, D, FW, NS> fs;
  if (EARLY) {
    fs.load_frags(wproj);
    if (c0 < c1) stage(0, c1 - 1);
    __syncthreads();
  }
  for (int c = c1 - 1; c >= c0; --c) {
    // This chunk's staging buffers.  Double-buffered, no store into them
    // needs a barrier of its own: the chunk that last read them (two back;
    // three back for K) is separated from the store by a dP barrier.
    const int step = c1 - 1 - c;
    const int par = NBUF == 2 ? step & 1 : 0, kp = step % NKB;
    IO* XQ = XQ2[par];
    IO* XK = XK2[kp];
    IO* XV = XV2[par];
    IO* XDO = XDO2[par];
    float (*GS)[2] = GS2[par];
    typename StX::Ssq* SSQ = SSQ2[par];
    typename StX::Ssq* SSK = SSK2[kp];
    const int tok0 = c * SH::CH;
    // this chunk's projection fragments (with early staging, issued at the
    // end of the previous chunk, before its dW' products)
    if (!EARLY) fs.load_frags(wproj);
    // With early staging this is the chunk's one barrier besides the dP
    // barrier: after it, every wave has finished the previous chunk's reads
    // of the other waves' LDS blocks (dP, dV partials, g shares), which this
    // chunk writes again before its dP barrier.
    if (EARLY) __syncthreads();
    // an earlier group's dK and dV of this chunk (rows past N read row N-1, unused)
    f32x4 old_k[ACC ? NDK : 1][ACC ? NTK : 1];
    float4 old_v[ACC ? SH::TT / QG : 1][ACC ? NIT : 1];
    if (ACC) {
#pragma unroll
      for (int kd = 0; kd < NDK; ++kd)
#pragma unroll
        for (int kt = 0; kt < NTK; ++kt) {
          const int dt = w % DT + kd * NW, tt = (DT < NW ? w / DT : 0) + kt * TT0STEP;
          const int tok = min(tok0 + tt * 16 + r, a.N - 1);
          if (dt < DT && tt < SH::TT)
            old_k[kd][kt] = *reinterpret_cast<const f32x4*>(dK + (size_t)tok * D + dt * 16 + 4 * g);
        }
#pragma unroll
      for (int q = 0; q < SH::TT / QG; ++q)
#pragma unroll
        for (int k = 0; k < NIT; ++k) {
          const int it = threadIdx.x + k * SH::NT;
          const int tok = min(tok0 + q * QG * 16 + it / C4, a.N - 1);
          if (it < QG * 16 * C4)
            old_v[q][k] = *reinterpret_cast<const float4*>(dV + (size_t)tok * SH::DV + 4 * (it % C4));
        }
    }
    if (!EARLY) {
      if (NBUF == 1) __syncthreads();   // single buffer: the previous chunk's reads are done
      stage(step, c);
      __syncthreads();
    }

    // phi(Q)/den as [token][feature] in the wave's LDS block: read back as it is
    // for the intra-chunk kernel matrix, transposed for the token sums (the
    // non-causal backward of K and V uses only the total R')
    if (CAUSAL) {
#pragma unroll
      for (int tt = 0; tt < SH::TT; ++tt) {
        ProjT<T> p[SH::PR];
        typename StX::Ssq ssq;
        project_tile_lds<T, D, FW, NS, StX::LD>(fs, XQ, SSQ, tt, p, ssq);
        const float sc = row_scale(ssq, inv_c, a.s_const, tok0 + tt * 16 + r < a.N) * GS[tt * 16 + r][0];
#pragma unroll
        for (int ft = 0; ft < SH::FT; ++ft)
          store_frag_nm<T>(PT[w], LDP, tt * 16, (2 * ft) * 16, (2 * ft + 1) * 16,
                           features<T, SH::FT, NS>(p, ft, sc, fv));
      }
    }
    // phi(K) and its P2-derivative fragments
    Frag<T> phk[SH::FT][SH::TT], psk[SH::FT][SH::TT];
#pragma unroll
    for (int tt = 0; tt < SH::TT; ++tt) {
      ProjT<T> p[SH::PR];
      typename StX::Ssq ssq;
      project_tile_lds<T, D, FW, NS, StX::LD>(fs, XK, SSK, tt, p, ssq);
      const float sc = row_scale(ssq, inv_c, a.s_const, tok0 + tt * 16 + r < a.N);
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) features_psi<T, SH::FT, NS>(p, ft, sc, phk[ft][tt], psk[ft][tt], fv);
    }
    // intra-chunk M[i][j] = dO_i . V_j - delta_i and A[i][j] = phi(Q_i)/den_i . phi(K_j), i >= j
    Frag<T> mp[CAUSAL ? SH::KT : 1][SH::TT], ap[CAUSAL ? SH::KT : 1][SH::TT];
    if (CAUSAL) {
#pragma unroll
      for (int tk = 0; tk < SH::TT; ++tk) {
        f32x4 m[SH::TT], at[SH::TT];
#pragma unroll
        for (int tq = 0; tq < SH::TT; ++tq) {
          m[tq] = zero4();
          at[tq] = zero4();
          if (tq >= tk) {
#pragma unroll
            for (int kd = 0; kd < SH::DV / 32; ++kd) {
              Frag<T> ao, bv;
              lds_row8(ao, XDO + (tq * 16 + r) * StV::LD, kd * 32 + 8 * g);
              lds_row8(bv, XV + (tk * 16 + r) * StV::LD, kd * 32 + 8 * g);
              mma(m[tq], ao, bv);
            }
#pragma unroll
            for (int ft = 0; ft < SH::FT; ++ft)
              mma(at[tq], load_frag_nm<T>(PT[w], LDP, tq * 16, (2 * ft) * 16, (2 * ft + 1) * 16), phk[ft][tk]);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const bool keep = tq > tk || 4 * g + i >= r;
              m[tq][i] = keep ? m[tq][i] - GS[tq * 16 + 4 * g + i][1] : 0.f;
              at[tq][i] = keep ? at[tq][i] : 0.f;
            }
          }
        }
#pragma unroll
        for (int ks = 0; ks < SH::KT; ++ks) {
          mp[ks][tk] = pair_tiles<T>(m[2 * ks], m[2 * ks + 1]);
          ap[ks][tk] = pair_tiles<T>(at[2 * ks], at[2 * ks + 1]);
        }
      }
    }
    // dphi(K)^T[feature][key] = phi(Q)^T M + R'^T-rows x [V | 1].  R' is
    // converted to operand fragments once per chunk and feature tile; the same
    // fragments, stored as [feature][value col], are the bf16 copy of R' that
    // the dV product reads back transposed.
    f32x4 dph[SH::FC][SH::TT];
    {
      Frag<T> vf[SH::TT][KG];
#pragma unroll
      for (int tk = 0; tk < SH::TT; ++tk)
#pragma unroll
        for (int kd = 0; kd < KG; ++kd) {
          if (32 * kd < SH::DV) {
            vf[tk][kd] = lds_tok_frag<T>(reinterpret_cast<const T*>(XV) + (tk * 16 + r) * StV::LD, kd);
          } else {
            Frag<T> f;
            f.zero();
            if (g == 0) { f.set(0, 1.0f); f.set(1, 1.0f); }
            vf[tk][kd] = f;
          }
        }
#pragma unroll
      for (int fc = 0; fc < SH::FC; ++fc) {
        Frag<T> rp[KG];
#pragma unroll
        for (int kd = 0; kd < KG; ++kd) {
          rp[kd] = pair_tiles<T>(RT[2 * kd][fc], 2 * kd + 1 < SH::DVT1 ? RT[2 * kd + 1][fc] : zero4());
          if (2 * kd + 1 < SH::DVT) {
            store_frag_nm<T>(RLw, RLP, fc * 16, (2 * kd) * 16, (2 * kd + 1) * 16, rp[kd]);
          } else if (2 * kd < SH::DVT) {
            store_tile_nm<T>(RLw, RLP, fc * 16, (2 * kd) * 16, RT[2 * kd][fc]);
          }
        }
#pragma unroll
        for (int tk = 0; tk < SH::TT; ++tk) {
          f32x4 acc = zero4();
          if (CAUSAL) {
#pragma unroll
            for (int ks = 0; ks < SH::KT; ++ks)
              if (32 * ks + 31 >= 16 * tk)
                mma(acc, lds_tr_frag<T>(PT[w], LDP, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, fc * 16), mp[ks][tk]);
          }
#pragma unroll
          for (int kd = 0; kd < KG; ++kd) mma(acc, rp[kd], vf[tk][kd]);
          dph[fc][tk] = acc;
        }
      }
    }
    // dV^T partial[value col][key] = dO^T A/den (intra) + R'[:dv]^T-rows x phi(K)
    f32x4 dvp[SH::DVT][SH::TT];
#pragma unroll
    for (int tk = 0; tk < SH::TT; ++tk)
#pragma unroll
      for (int dt = 0; dt < SH::DVT; ++dt) {
        f32x4 acc = zero4();
        if (CAUSAL) {
#pragma unroll
          for (int ks = 0; ks < SH::KT; ++ks)
            if (32 * ks + 31 >= 16 * tk) mma(acc, lds_tr_frag<T>(reinterpret_cast<const T*>(XDO), StV::LD, 32 * ks + 4 * g, 32 * ks + 16 + 4 * g, dt * 16), ap[ks][tk]);
        }
#pragma unroll
        for (int ft = 0; ft < SH::FT; ++ft)
          mma(acc, lds_tr_frag<T>(RLw, RLP, (2 * ft) * 16 + 4 * g, (2 * ft + 1) * 16 + 4 * g, dt * 16),
              phk[ft][tk]);
        dvp[dt][tk] = acc;
      }
    // dV: reduce the per-wave partials.  With one reduction round per chunk the
    // partials are written now and reduced after the dP barrier below, which
    // orders these writes before every wave's reads (the slots are written
    // again only after the next chunk's staging barrier); with several rounds
    // each round has barriers of its own.
    constexpr bool DEFER_DV = QG == SH::TT;
    auto dv_write = [&](int q0) {
#pragma unroll
      for (int qq = 0; qq < QG; ++qq)
#pragma unroll
        for (int dt = 0; dt < SH::DVT; ++dt)
          *reinterpret_cast<f32x4*>(&RED(w)[qq * 16 + r][dt * 16 + 4 * g]) = dvp[dt][q0 + qq];
    };
    auto dv_reduce = [&](int q0) {
#pragma unroll
      for (int k = 0; k < NIT; ++k) {
        const int it = threadIdx.x + k * SH::NT;
        if (it >= QG * 16 * C4) break;
        const int t = it / C4, c4 = it % C4;
        const int tok = tok0 + q0 * 16 + t;
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ACC) s = old_v[q0 / QG][k];   // later frequency groups add their share
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
          const float4 v = *reinterpret_cast<const float4*>(&RED(ww)[t][4 * c4]);
          s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
        if (tok < a.N) *reinterpret_cast<float4*>(dV + (size_t)tok * SH::DV + 4 * c4) = s;
      }
    };
    if (DEFER_DV) {
      dv_write(0);
    } else {
#pragma unroll
      for (int q0 = 0; q0 < SH::TT; q0 += QG) {
        if (q0 > 0) __syncthreads();   // the previous round's reads of every slot are done
        dv_write(q0);
        __syncthreads();
        dv_reduce(q0);
      }
    }
    // R'^T += [dO | -delta]^T-rows x phi(Q)/den  (after every use of R'_{>c})
    if (CAUSAL) {
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
    // chain rule through phi(K)
    f32x4 dp[SH::PR][SH::TT];
    float gp[SH::TT];
#pragma unroll
    for (int tt = 0; tt < SH::TT; ++tt) {
      float gs = 0.f;
#pragma unroll
      for (int ft = 0; ft < SH::FT; ++ft) {
        f32x4 d2 = zero4();
        gs += feature_grad<T, SH::FT, NS>(phk[ft][tt], psk[ft][tt], dph[2 * ft][tt], dph[2 * ft + 1][tt], dp[ft][tt], d2);
        if (NS) dp[SH::FT + ft][tt] = d2;
      }
      gp[tt] = gs;   // this lane group's share; the four shares are summed in the dK reduction
    }
    // dK = dP W' over all projection rows + (2/c) g k, g = <phi(K), dphi(K)>;
    // dtau -= g ||k||^2 / c.  Each wave computes whole output tiles (d tile,
    // token tile) from every wave's dP block and that wave's dX fragments, so
    // no cross-wave reduction is needed.  Wave w takes the d tiles
    // dt = w mod DT (+ NW, ...) and, when there are fewer d tiles than waves,
    // the token tiles tt = w / DT (+ NW / DT, ...).  The dX fragments of its
    // first d tile are loaded before the barrier, so their latency overlaps it.
    if (!HOLD_WF) load_wf(w % DT);
    // the next chunk's rows (the last step stages its own rows again, unused)
    if (EARLY) stage(step + 1, c - 1 >= c0 ? c - 1 : c);
    // dP of this wave as [token][projection row] in its LDS block (its own reads
    // of phi(Q)/den there are done: one wave's LDS accesses complete in order),
    // and this lane's share of g per token
#pragma unroll
    for (int pr = 0; pr < SH::PR; ++pr)
#pragma unroll
      for (int tt = 0; tt < SH::TT; ++tt) store_tile_nm<T>(PT[w], LDP, tt * 16, pr * 16, dp[pr][tt]);
#pragma unroll
    for (int tt = 0; tt < SH::TT; ++tt) GP[tt * 16 + r][w][g] = gp[tt];
    __syncthreads();   // every wave's dP block and g shares complete
    if (DEFER_DV) dv_reduce(0);
#pragma unroll
    for (int kd = 0; kd < NDK; ++kd) {
      const int dt = w % DT + kd * NW;
      if (dt >= DT) break;
      f32x4 acc[NTK];
#pragma unroll
      for (int kt = 0; kt < NTK; ++kt) {
        const int tt = (DT < NW ? w / DT : 0) + kt * TT0STEP;
        acc[kt] = zero4();
        if (tt >= SH::TT) continue;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
#pragma unroll
          for (int ks = 0; ks < WTS::KP; ++ks) {
            Frag<T> b = load_frag_nm<T>(PT[ww], LDP, tt * 16, (2 * ks) * 16, (2 * ks + 1) * 16);
            if (2 * ks + 1 >= SH::PR) {   // no second row tile: keep unwritten LDS out of the product
#pragma unroll
              for (int j = 4; j < 8; ++j) b.set(j, 0.f);
            }
#pragma unroll
            for (int sp = 0; sp < WTS::NSPLIT; ++sp) mma(acc[kt], wf[ww][ks][sp], b);
          }
        }
      }
      // the next d tile's dX fragments, issued ahead of this tile's stores so
      // that waiting for them does not wait for the stores
      if (kd + 1 < NDK && dt + NW < DT) load_wf(dt + NW);
#pragma unroll
      for (int kt = 0; kt < NTK; ++kt) {
        const int tt = (DT < NW ? w / DT : 0) + kt * TT0STEP;
        if (tt >= SH::TT) continue;
        const int tl = tt * 16 + r, tok = tok0 + tl;
        float gg = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
          const float4 v = *reinterpret_cast<const float4*>(&GP[tl][ww][0]);
          gg += (v.x + v.y) + (v.z + v.w);
        }
        if (tok < a.N) {
          const float k2 = 2.0f * inv_c * gg;
          const IO* kr = XK + tl * StX::LD + dt * 16 + 4 * g;
          f32x4 s;
#pragma unroll
          for (int i = 0; i < 4; ++i) s[i] = acc[kt][i] + k2 * io_to_float(kr[i]);
          if (ACC) s += old_k[kd][kt];   // later frequency groups add their share
          *reinterpret_cast<f32x4*>(dK + (size_t)tok * D + dt * 16 + 4 * g) = s;
          if (dt == 0 && g == 0) dtau_acc -= gg * SSK[tl] * inv_c;
        }
      }
    }
    if (EARLY) fs.load_frags(wproj);   // the next chunk's (the last step's are unused)
    {
      // one 32-token k-step per chunk, added to the LDS partial one
      // projection-row tile at a time
      static_assert(SH::KT == 1, "one token k-step per chunk");
      Frag<T> xk[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) xk[dt] = lds_tr_frag<T>(reinterpret_cast<const T*>(XK), StX::LD, 4 * g, 16 + 4 * g, dt * 16);
#pragma unroll
      for (int pr = 0; pr < SH::PR; ++pr) {
        const Frag<T> dpt = lds_tr_frag<T>(PT[w], LDP, 4 * g, 16 + 4 * g, pr * 16);
        dw_mma_row<D, T>(DWL[w], pr, dpt, xk);
      }
    }
  }
  const size_t nmat = NS ? 2 : 1;
  float* out = a.dwpart + (((size_t)1 * a.BH + bh) * a.segments + seg) * nmat * SH::M * D;
  dump_dw<SH, D, FW, NS>(out, DWL[w], w * FW);
  // dtau partial of this workgroup: fixed-order tree sum
  TRED[threadIdx.x] = dtau_acc;
  __syncthreads();
  for (int s = SH::NT / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) TRED[threadIdx.x] += TRED[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) a.dtaupart[(size_t)bh * a.segments + seg] = TRED[0];
}

// ---------------------------------------------------------------------------
// Fixed-order reduction of the frequency-gradient and dtau partials.
// dwpart: [2][B*H][P][nmat][m][d]; the key side's blocks hold the sums of
// both sides in [matrix][m][d] order.  dW'1, dW'2 -> dW1 = (dW'1+dW'2)/2,
// dW2 = (dW'1-dW'2)/2 because W'1 = (W1+W2)/2 and W'2 = (W1-W2)/2.
// ---------------------------------------------------------------------------
template <int NMAT>
__global__ __launch_bounds__(256) void k_bwd_reduce(BwdArgs a, int md4, int d) {
  // 256 elements (f, k) of one head per workgroup, 4 consecutive per thread;
  // the 4 waves split the list of partials (b, segment; each already the sum
  // of the query and key sides) round-robin and
  // issue a batch of loads of every matrix before summing it (a partial past
  // the list reads the last one, added as zero), then the 4 wave sums are
  // combined in a fixed order.
  constexpr int BATCH = 8;
  __shared__ float4 part[NMAT][4][64];
  const int e4 = blockIdx.x * 64 + (threadIdx.x % 64);
  const int q = threadIdx.x / 64;
  const int h = blockIdx.y;
  const int count = a.B * a.segments;
  const float4* src = reinterpret_cast<const float4*>(a.dwpart);
  float4 acc[NMAT];
#pragma unroll
  for (int mat = 0; mat < NMAT; ++mat) acc[mat] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (e4 < md4) {
    for (int i0 = q; i0 < count; i0 += 4 * BATCH) {
      float4 v[BATCH][NMAT];
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const int j = min(i0 + 4 * u, count - 1);
        const int b = j / a.segments, p = j % a.segments;
        const size_t blk = ((size_t)1 * a.BH + (size_t)b * a.H + h) * a.segments + p;
#pragma unroll
        for (int mat = 0; mat < NMAT; ++mat) v[u][mat] = src[(blk * NMAT + mat) * md4 + e4];
      }
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const float k = i0 + 4 * u < count ? 1.f : 0.f;
#pragma unroll
        for (int mat = 0; mat < NMAT; ++mat) {
          acc[mat].x += k * v[u][mat].x; acc[mat].y += k * v[u][mat].y;
          acc[mat].z += k * v[u][mat].z; acc[mat].w += k * v[u][mat].w;
        }
      }
    }
  }
#pragma unroll
  for (int mat = 0; mat < NMAT; ++mat) part[mat][q][threadIdx.x % 64] = acc[mat];
  __syncthreads();
  if (q == 0 && e4 < md4) {
    const int t = threadIdx.x;
    float4 x[NMAT];
#pragma unroll
    for (int mat = 0; mat < NMAT; ++mat) {
      const float4 p0 = part[mat][0][t], p1 = part[mat][1][t], p2 = part[mat][2][t], p3 = part[mat][3][t];
      x[mat] = make_float4((p0.x + p1.x) + (p2.x + p3.x), (p0.y + p1.y) + (p2.y + p3.y),
                           (p0.z + p1.z) + (p2.z + p3.z), (p0.w + p1.w) + (p2.w + p3.w));
    }
    float4* o1 = reinterpret_cast<float4*>(a.dW1 + (size_t)h * a.dw_stride) + e4;
    if (4 * e4 / d >= a.fvalid) {
      // a padding row of a last frequency group: no output row
    } else if (NMAT == 2) {
      float4* o2 = reinterpret_cast<float4*>(a.dW2 + (size_t)h * a.dw_stride) + e4;
      const float4 u = x[0], w = x[NMAT - 1];
      *o1 = make_float4(0.5f * (u.x + w.x), 0.5f * (u.y + w.y), 0.5f * (u.z + w.z), 0.5f * (u.w + w.w));
      *o2 = make_float4(0.5f * (u.x - w.x), 0.5f * (u.y - w.y), 0.5f * (u.z - w.z), 0.5f * (u.w - w.w));
    } else {
      *o1 = x[0];
    }
  }
  if (a.dtau && blockIdx.x == 0 && threadIdx.x == 0) {
    float s = 0.f;
    for (int b = 0; b < a.B; ++b)
      for (int p = 0; p < a.segments; ++p) s += a.dtaupart[((size_t)b * a.H + h) * a.segments + p];
    a.dtau[h] = a.acc ? a.dtau[h] + s : s;
  }
}

// ---------------------------------------------------------------------------
// Host-side dispatch.
// ---------------------------------------------------------------------------
// Frequencies per wave (FW) and waves per workgroup (NW) of the pre-pass and
// the dQ sweep (A) and of the dK/dV sweep (B).  The states, the partial sums
// and the per-token scalars have split-independent layouts; each split has its
// own prepared fragments.
template <class T, int D, bool NS, int FWA, int NWA, int FWB, int NWB>
static hipError_t run_bwd_t(const BwdArgs& a, bool causal, hipStream_t st) {
  typedef Shape<T, D, FWA, NWA, NS, BWD_CHUNK> SA;
  typedef Shape<T, D, FWB, NWB, NS, BWD_CHUNK> SB;
  static_assert(SA::M == SB::M && SA::STATE == SB::STATE, "splits of one shape");
  const dim3 grid(a.segments * a.BH);
  if (a.wfrag_kv != a.wfrag)   // both splits' fragments in one launch
    k_prep_freqs2<T, D, FWA, NWA, FWB, NWB, NS><<<dim3(a.H, NWA > NWB ? NWA : NWB, 4), WAVE, 0, st>>>(
        a.W1, a.W2, a.wfrag, a.wfrag_kv, a.w_stride);
  else
    k_prep_freqs<T, D, FWA, NWA, NS><<<dim3(a.H, NWA, 2), WAVE, 0, st>>>(a.W1, a.W2, a.wfrag, a.w_stride);
  // With the forward's key-side states passed in, the dQ sweep does the
  // pre-pass's query-side work itself and no pre-pass runs; the R' local
  // states it leaves feed the scan, or the dK/dV sweep's own suffix sum.
  const bool wr = a.fstate != nullptr;
  // a padded frequency group (only the 64-frequency shape has one, and it runs
  // first, so it never adds) takes the masking kernel variants
  const bool masked = a.fvalid < SA::M;
  constexpr bool CAN_MASK = SA::M == 64;
  if (masked && (!CAN_MASK || a.acc)) return hipErrorInvalidValue;
  auto scan_r = [&]() -> hipError_t {
    if (causal && a.rfold) return hipSuccess;
    return launch_state_scan(a.fstate ? nullptr : a.sstate, a.rstate, a.BH, a.segments, 1, SA::STATE, causal, st,
                             a.segments);
  };
  if (!wr) {
    timing_mark(KC_BWD_PREPASS, st, true);
    if constexpr (CAN_MASK) {
      if (masked) {
        if (a.fstate) k_bwd_prepass<T, D, FWA, NWA, NS, false, true><<<grid, SA::NT, 0, st>>>(a);
        else k_bwd_prepass<T, D, FWA, NWA, NS, true, true><<<grid, SA::NT, 0, st>>>(a);
      }
    }
    if (!masked) {
      if (a.fstate) k_bwd_prepass<T, D, FWA, NWA, NS, false><<<grid, SA::NT, 0, st>>>(a);
      else k_bwd_prepass<T, D, FWA, NWA, NS, true><<<grid, SA::NT, 0, st>>>(a);
    }
    timing_mark(KC_BWD_PREPASS, st, false);
    const hipError_t e = scan_r();
    if (e != hipSuccess) return e;
  }
  timing_mark(KC_BWD_DQ, st, true);
  // a later frequency group adds into the earlier groups' outputs
  {
    const hipError_t e = launch_bwd_dq<T, D, FWA, NWA, NS>(a, causal, a.acc != 0, wr, masked, st);
    if (e != hipSuccess) return e;
  }
  timing_mark(KC_BWD_DQ, st, false);
  if (wr) {
    const hipError_t e = scan_r();
    if (e != hipSuccess) return e;
  }
  timing_mark(KC_BWD_DKV, st, true);
  if (a.acc) {
    if (causal)
      k_bwd_dkv<T, D, FWB, NWB, NS, true, true><<<grid, SB::NT, 0, st>>>(a);
    else
      k_bwd_dkv<T, D, FWB, NWB, NS, false, true><<<grid, SB::NT, 0, st>>>(a);
  } else if (masked) {
    if constexpr (CAN_MASK) {
      if (causal)
        k_bwd_dkv<T, D, FWB, NWB, NS, true, false, true><<<grid, SB::NT, 0, st>>>(a);
      else
        k_bwd_dkv<T, D, FWB, NWB, NS, false, false, true><<<grid, SB::NT, 0, st>>>(a);
    }
  } else {
    if (causal)
      k_bwd_dkv<T, D, FWB, NWB, NS, true, false><<<grid, SB::NT, 0, st>>>(a);
    else
      k_bwd_dkv<T, D, FWB, NWB, NS, false, false><<<grid, SB::NT, 0, st>>>(a);
  }
  timing_mark(KC_BWD_DKV, st, false);
  static_assert((SA::M * D) % 4 == 0, "the reduce moves 4 floats per thread");
  constexpr int MD4 = SA::M * D / 4;
  dim3 rgrid((MD4 + 63) / 64, a.H);
  timing_mark(KC_BWD_REDUCE, st, true);
  k_bwd_reduce<NS ? 2 : 1><<<rgrid, 256, 0, st>>>(a, MD4, D);
  timing_mark(KC_BWD_REDUCE, st, false);
  return hipGetLastError();
}

template <class T, int D, int FWA, int NWA, int FWB, int NWB>
static hipError_t run_bwd_v(const BwdArgs& a, bool ns, bool causal, hipStream_t st) {
  return ns ? run_bwd_t<T, D, true, FWA, NWA, FWB, NWB>(a, causal, st)
            : run_bwd_t<T, D, false, FWA, NWA, FWB, NWB>(a, causal, st);
}

hipError_t launch_bwd(const BwdArgs& a, const KernelShape& ks, hipStream_t st) {
  if (ks.bf16) {
    if (ks.d == 32 && ks.m == 64) return run_bwd_v<__bf16, 32, 16, 4, 16, 4>(a, ks.nonstationary, ks.causal, st);
    if (ks.d == 64 && ks.m == 64) return run_bwd_v<__bf16, 64, 16, 4, 16, 4>(a, ks.nonstationary, ks.causal, st);
    if (ks.d == 64 && ks.m == 128) return run_bwd_v<__bf16, 64, 16, 8, 32, 4>(a, ks.nonstationary, ks.causal, st);
    if (ks.d == 128 && ks.m == 64) return run_bwd_v<__bf16, 128, 16, 4, 16, 4>(a, ks.nonstationary, ks.causal, st);
  } else {
    if (ks.d == 32 && ks.m == 64) return run_bwd_v<float, 32, 16, 4, 16, 4>(a, ks.nonstationary, ks.causal, st);
  }
  return hipErrorNotSupported;
}

// Whether the dK/dV sweep splits the frequencies differently from the other
// backward kernels (then it needs a second block of prepared fragments).
bool bwd_split_differs(const KernelShape& ks) { return ks.bf16 && ks.d == 64 && ks.m == 128; }

size_t bwd_state_floats(const KernelShape& ks) { return fwd_state_floats(ks); }
// both sides (query rows and key rows) of the frequency-gradient partials
size_t bwd_dw_floats(const KernelShape& ks) {
  return (size_t)2 * (ks.nonstationary ? 2 : 1) * ks.m * ks.d;
}

}  // namespace flex
