// C ABI of the RFF linear attention library: argument validation, workspace
// sizing, segment selection and dispatch to the gfx950 kernels.
#include "../../include/flex.h"
#include "flex_kernels.hpp"

#include <math.h>
#include <string.h>

#include <mutex>
#include <vector>

using namespace flex;

namespace {

constexpr int kChunk = 64;
constexpr int kCUs = 256;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Chunk lengths of the causal forward sweep.  The segment split, the state
// pre-pass and the non-causal sweep work in 64-token chunks whatever the
// chunk; the backward in 32-token chunks.
bool chunk_supported(int c) { return c == 0 || c == 16 || c == 32 || c == 64; }
int chunk_of(const flex_desc* d) { return d->chunk == 0 ? kChunk : d->chunk; }

// Attention shapes: d and dv in {32, 64, 128} for bf16 (d = dv = 32 for fp32),
// m a multiple of 16 up to 256.  Shapes that no single kernel covers run as
// frequency groups (groups_of); dv != d runs at the wider of the two on
// zero-padded operands (padded_desc).
bool shape_supported(const flex_desc* d) {
  if (d->dv != d->d && (d->io_dtype != FLEX_BF16 || !(d->dv == 32 || d->dv == 64 || d->dv == 128)))
    return false;
  if (d->grad_dtype != FLEX_F32) return false;
  if (!chunk_supported(d->chunk)) return false;
  if (d->m % 16 != 0 || d->m > 256) return false;
  if (d->io_dtype == FLEX_BF16) return d->d == 32 || d->d == 64 || d->d == 128;
  return d->d == 32;
}

// Shapes of the standalone feature map: the attention's d and m (it ignores
// dv).  It runs in slices of the frequency count of its kernel for d
// (fmap_slice_m), the last one partly filled when that does not divide m.
bool fmap_shape_supported(const flex_desc* d) {
  if (d->m % 16 != 0 || d->m > 256) return false;
  if (d->io_dtype == FLEX_BF16) return d->d == 32 || d->d == 64 || d->d == 128;
  return d->d == 32;
}
int fmap_slice_m(const flex_desc* d) {
  if (d->d == 128) return 256;
  if (d->d == 64) return d->m <= 64 ? 64 : 128;
  return 64;
}

// 0 = ok, else a flex_status: the descriptor's fields, without the shape list
int32_t check_desc_fields(const flex_desc* d) {
  if (!d) return FLEX_ERR_INVALID_ARG;
  if (d->B <= 0 || d->H <= 0 || d->N <= 0 || d->d <= 0 || d->dv <= 0 || d->m <= 0)
    return FLEX_ERR_INVALID_ARG;
  if (d->variant != FLEX_STATIONARY && d->variant != FLEX_NONSTATIONARY) return FLEX_ERR_INVALID_ARG;
  if (d->causal != 0 && d->causal != 1) return FLEX_ERR_INVALID_ARG;
  if (d->io_dtype != FLEX_F32 && d->io_dtype != FLEX_BF16) return FLEX_ERR_INVALID_ARG;
  if (d->grad_dtype != FLEX_F32 && d->grad_dtype != FLEX_BF16) return FLEX_ERR_INVALID_ARG;
  if (d->chunk < 0 || d->segments < 0) return FLEX_ERR_INVALID_ARG;
  if (!(d->sigma > 0.0f) || !isfinite(d->sigma)) return FLEX_ERR_INVALID_ARG;
  // element counts must fit the 32-bit token and 64-bit element indexing used on device
  const long long bhn = (long long)d->B * d->H * d->N;
  if (bhn > (1LL << 40) || (long long)d->B * d->H > (1LL << 30)) return FLEX_ERR_INVALID_ARG;
  return FLEX_OK;
}

// 0 = ok, else a flex_status
int32_t check_desc(const flex_desc* d) {
  const int32_t st = check_desc_fields(d);
  if (st != FLEX_OK) return st;
  if (!shape_supported(d)) return FLEX_ERR_UNSUPPORTED;
  return FLEX_OK;
}

// The feature map ignores dv, causal, chunk, segments and grad_dtype: the
// descriptor is checked with those fields set to values every shape accepts.
int32_t check_fmap_desc(const flex_desc* d) {
  if (!d) return FLEX_ERR_INVALID_ARG;
  flex_desc c = *d;
  c.dv = c.d;
  c.causal = 0;
  c.chunk = 0;
  c.segments = 0;
  c.grad_dtype = FLEX_F32;
  const int32_t st = check_desc_fields(&c);
  if (st != FLEX_OK) return st;
  return fmap_shape_supported(&c) ? FLEX_OK : FLEX_ERR_UNSUPPORTED;
}

// Shapes of the decode step (one generic kernel): d and dv multiples of 4 up
// to 128; up to 1024 frequencies.
bool decode_supported(const flex_desc* d) {
  return d->d % 4 == 0 && d->d <= 128 && d->dv % 4 == 0 && d->dv <= 128 && d->m <= 1024 &&
         d->grad_dtype == FLEX_F32;
}

KernelShape kshape(const flex_desc* d) {
  KernelShape k;
  k.bf16 = d->io_dtype == FLEX_BF16;
  k.nonstationary = d->variant == FLEX_NONSTATIONARY;
  k.causal = d->causal != 0;
  k.d = d->d;
  k.m = d->m;
  return k;
}

// Frequency groups of the attention kernels.  The kernels cover (d, m) =
// (32, 64), (64, 64), (64, 128) (bf16) and (128, 64) in one launch per pass;
// every other shape runs as groups of 128 frequencies (bf16 d = 64, m a
// multiple of 128) or of 64 (at d = 128, m = 256 the per-workgroup state and
// frequency-gradient partials of one group fit registers and LDS, all 256
// frequencies would not).  When 64 does not divide m, the first group holds
// the first `last` frequencies and zero rows after them, whose features the
// kernels mask to zero (it runs first, so only write variants need masking).
// The groups' contributions to the numerator, denominator and the Q/K/V/tau
// gradients are summed in launch order; the frequency gradients of a group
// are its own rows.
struct Groups {
  int n, m, last;
};
Groups groups_of(const flex_desc* d) {
  if (d->d == 64 && d->m % 128 == 0 && d->io_dtype == FLEX_BF16) return Groups{d->m / 128, 128, 128};
  const int n = (d->m + 63) / 64;
  return Groups{n, 64, d->m - 64 * (n - 1)};
}

// First frequency row of group g (the padded group, if any, is group 0).
int group_off(const Groups& G, int g) { return g == 0 ? 0 : G.last + (g - 1) * G.m; }

// Padded frequency rows of a first group that 64 does not fill: [H][group][d]
// per matrix, at the end of the forward and backward workspaces.
size_t pad_bytes(const flex_desc* d) {
  const Groups G = groups_of(d);
  if (G.last == G.m) return 0;
  const size_t nmat = d->variant == FLEX_NONSTATIONARY ? 2 : 1;
  return nmat * align256((size_t)d->H * G.m * d->d * sizeof(float));
}

// The padded rows' place in a workspace that ends at `end`.
struct PadRows {
  float* w1;
  float* w2;
};
PadRows pad_rows_of(const flex_desc* d, char* end) {
  const size_t pb = pad_bytes(d);
  if (pb == 0) return PadRows{nullptr, nullptr};
  char* p = end - pb;
  const size_t one = align256((size_t)d->H * groups_of(d).m * d->d * sizeof(float));
  return PadRows{reinterpret_cast<float*>(p),
                 d->variant == FLEX_NONSTATIONARY ? reinterpret_cast<float*>(p + one) : nullptr};
}

// Frequency rows of group g: the caller's rows of W1/W2 (head stride m d),
// or for a padded group a zero-padded copy of them (head stride group width
// x d), written on the stream first.  fvalid: the group's rows that are
// frequencies.  False if the copy's launch fails.
bool group_rows(const flex_desc* d, const Groups& G, const PadRows& pr, int g, const float* W1, const float* W2,
                hipStream_t st, const float** w1, const float** w2, int* stride, int* fvalid) {
  const size_t woff = (size_t)group_off(G, g) * d->d;
  const bool padded = g == 0 && G.last < G.m;
  *fvalid = g == 0 ? G.last : G.m;
  if (!padded) {
    *w1 = W1 + woff;
    *w2 = W2 ? W2 + woff : nullptr;
    *stride = d->m * d->d;
    return true;
  }
  if (launch_pad_rows(W1 + woff, pr.w1, d->H, G.last, G.m, d->d, d->m * d->d, st) != hipSuccess) return false;
  if (W2 && launch_pad_rows(W2 + woff, pr.w2, d->H, G.last, G.m, d->d, d->m * d->d, st) != hipSuccess) return false;
  *w1 = pr.w1;
  *w2 = W2 ? pr.w2 : nullptr;
  *stride = G.m * d->d;
  return true;
}

// Kernel shape of the attention passes (one frequency group).
KernelShape attn_shape(const flex_desc* d) {
  KernelShape k = kshape(d);
  k.m = groups_of(d).m;
  return k;
}

int nchunks_of(const flex_desc* d) { return (d->N + kChunk - 1) / kChunk; }

// Chunks per workgroup of the non-causal sweep (its chunks are independent).
constexpr int kSweepChunks = 8;
// The bf16 stationary shapes with m = 64 read out with the tokens split
// across waves (k_fwd_readout): a workgroup holds the whole total state, so it
// takes up to 64 chunks, about one round of two workgroups per CU.
constexpr int kReadoutChunks = 64;
bool readout_split(const flex_desc* d) {
  return !d->causal && d->io_dtype == FLEX_BF16 && d->variant == FLEX_STATIONARY && d->m == 64 && d->d <= 64;
}

// Segments whose local state the forward pre-pass forms: a causal forward
// reads only exclusive prefixes, so the last segment's own state is never used.
int pre_segs_of(const flex_desc* d, int P) { return d->causal ? P - 1 : P; }

// Forward state pre-pass workgroups per segment (sub-segments): 1, 2, 4 or 8,
// dividing the segment's chunks.  More sub-segments shorten the pre-pass's
// critical path when its workgroups underfill the CUs (fwd_state_wgs_per_cu
// workgroups per CU at a time) but write and scan more states; the
// cost is the rounds of chunks (about a third of a sweep chunk each, scaled
// by MFMA work like pick_segments) plus that state traffic at 5 TB/s.
int fwd_sub_of(const flex_desc* d, int P) {
  const int nc = nchunks_of(d);
  const int cps = (nc + P - 1) / P;
  const long long used = pre_segs_of(d, P);
  if (used <= 0) return 1;
  const KernelShape ks = attn_shape(d);
  const long long cap = (long long)kCUs * fwd_state_wgs_per_cu(ks);
  const double m_eff = ks.nonstationary ? 2.0 * ks.m : ks.m;
  const double t_pre = 2.2e-6 * (2.0 * ks.d * m_eff + 4.0 * ks.m * (d->dv + 1)) / 66048.0;
  const double state_bytes = (double)fwd_state_floats(ks) * sizeof(float);
  int best = 1;
  double best_t = 1e30;
  for (int sub = 1; sub <= 8; sub *= 2) {
    if (cps % sub != 0) break;
    const long long wgs = (long long)d->B * d->H * used * sub;
    const double t = (double)((wgs + cap - 1) / cap) * (cps / sub) * t_pre + 2.0 * wgs * state_bytes / 5.0e12;
    if (t < best_t - 1e-12) { best_t = t; best = sub; }
  }
  return best;
}

// Whether the causal sweeps (the forward's and the backward's dQ sweep) sum
// their carry-in from the segments' local states themselves, with no scan
// launch: when a workgroup reads at most kFoldMax local states.  The sum runs
// in the scan's order, so both ways give the same bits.
constexpr int kFoldMax = 4;
constexpr int kRFoldMax = 8;   // R' suffixes: native-layout reads, cheaper to sum
int fwd_fold_of(const flex_desc* d, int P) {
  return d->causal && (long long)pre_segs_of(d, P) * fwd_sub_of(d, P) <= kFoldMax ? 1 : 0;
}

// Segments per (b,h): enough workgroups to cover the 256 CUs in whole rounds
// while keeping the per-segment state traffic small.  Costs are in units of
// one sweep chunk: the sweep's rounds of chunks (a pre-pass adds about a third
// of a chunk), the hand-off, and the segment states' HBM traffic (written by
// the pre-pass, read and written by the scan, read by the sweep).  A chunk's
// time is estimated from its MFMA work relative to the d = 64, m = 128
// nonstationary shape, measured at about 6.7 us per 64-token chunk.
int pick_segments(const flex_desc* d) {
  const int nc = nchunks_of(d);
  if (d->segments > 0) return d->segments < nc ? d->segments : nc;
  const long long bh = (long long)d->B * d->H;
  const KernelShape ks = attn_shape(d);
  const double m_eff = ks.nonstationary ? 2.0 * ks.m : ks.m;
  const double work = 2.0 * ks.d * m_eff + 4.0 * ks.m * (d->dv + 1);   // MFMA flop per token
  const double t_chunk = 6.7e-6 * work / 66048.0;
  const double state_bytes = (double)fwd_state_floats(ks) * sizeof(float);
  int best = 1;
  double best_cost = 1e30;
  for (int p = 1; p <= nc && p <= kCUs; ++p) {
    const int cps = (nc + p - 1) / p;
    const int used = (nc + cps - 1) / cps;  // segments that hold chunks
    if (used != p) continue;
    const long long wgs = bh * p;
    const long long rounds = (wgs + kCUs - 1) / kCUs;
    const double traffic = 4.0 * p * bh * state_bytes / 5.0e12 / t_chunk;
    const double cost = rounds * (double)cps * (p > 1 || !d->causal ? 1.35 : 1.0) + 0.5 * p * bh / kCUs + traffic;
    if (cost < best_cost - 1e-9) { best_cost = cost; best = p; }
  }
  return best;
}

float s_const_of(const flex_desc* d) {
  const double s = d->variant == FLEX_STATIONARY ? d->sigma / sqrt((double)d->m)
                                                 : d->sigma / (2.0 * sqrt((double)d->m));
  return (float)s;
}


// Forward workspace: the segment states of every frequency group, one block of
// prepared fragments (reused group after group) and, with several groups, the
// fp32 numerator / denominator sums.
size_t fwd_group_state_bytes(const flex_desc* d) {
  const size_t P = (size_t)pick_segments(d);
  return align256((size_t)d->B * d->H * P * fwd_sub_of(d, (int)P) * fwd_state_floats(attn_shape(d)) *
                  sizeof(float));
}
size_t fwd_acc_bytes(const flex_desc* d) {
  if (groups_of(d).n == 1) return 0;
  const size_t rows = (size_t)d->B * d->H * d->N;
  return align256(rows * d->dv * sizeof(float)) + align256(rows * sizeof(float));
}

// dv != d: the attention runs at width w = max(d, dv) on zero-padded
// operands.  With dv > d, Q, K and the frequency rows get w - d zero columns:
// the projections W x and the norms |x|^2 are unchanged, and the padded
// columns of dQ, dK and dW come out zero and are dropped.  With dv < d, V, O
// and dO get d - dv zero columns: den, delta and every gradient but the
// padded columns of dV are unchanged.  The padded copies sit after the
// padded shape's own workspace.
flex_desc padded_desc(const flex_desc* d) {
  flex_desc p = *d;
  p.d = p.dv = d->d > d->dv ? d->d : d->dv;
  return p;
}
struct ValuePad {
  size_t q, k, w1, w2, dq, dk, dw1, dw2, v, o, dO, dv, total;
};
ValuePad value_pad_of(const flex_desc* d, int pass) {
  ValuePad L;
  memset(&L, 0, sizeof(L));
  if (d->dv == d->d) return L;
  const size_t rows = (size_t)d->B * d->H * d->N, hm = (size_t)d->H * d->m;
  const size_t w = d->d > d->dv ? d->d : d->dv;
  const size_t io = d->io_dtype == FLEX_BF16 ? 2 : 4;
  const bool ns = d->variant == FLEX_NONSTATIONARY;
  const bool bwd = pass == FLEX_PASS_BWD;
  size_t off = 0;
  if (d->dv > d->d) {
    L.q = off;  off += align256(rows * w * io);
    L.k = off;  off += align256(rows * w * io);
    L.w1 = off; off += align256(hm * w * sizeof(float));
    if (ns) { L.w2 = off; off += align256(hm * w * sizeof(float)); }
    if (bwd) {
      L.dq = off;  off += align256(rows * w * sizeof(float));
      L.dk = off;  off += align256(rows * w * sizeof(float));
      L.dw1 = off; off += align256(hm * w * sizeof(float));
      if (ns) { L.dw2 = off; off += align256(hm * w * sizeof(float)); }
    }
  } else {
    L.v = off; off += align256(rows * w * io);
    L.o = off; off += align256(rows * w * io);
    if (bwd) {
      L.dO = off; off += align256(rows * w * io);
      L.dv = off; off += align256(rows * w * sizeof(float));
    }
  }
  L.total = off;
  return L;
}

size_t ws_bytes_of(const flex_desc* d, int pass) {
  if (d->dv != d->d && pass != FLEX_PASS_FEATURE_MAP) {
    const flex_desc pd = padded_desc(d);
    return ws_bytes_of(&pd, pass) + value_pad_of(d, pass).total;
  }
  const KernelShape ks = attn_shape(d);
  const size_t bh = (size_t)d->B * d->H;
  const size_t P = (size_t)pick_segments(d);
  if (pass == FLEX_PASS_FEATURE_MAP) return 0;
  const size_t wf = align256(wfrag_bytes(ks, d->H));
  if (pass == FLEX_PASS_FWD) return groups_of(d).n * fwd_group_state_bytes(d) + wf + fwd_acc_bytes(d) + pad_bytes(d);
  // backward: key-side and query-side states, per-token scalars, frequency-gradient
  // and dtau partials
  return 2 * align256(bh * P * bwd_state_floats(ks) * sizeof(float)) +
         align256(bh * (size_t)d->N * 2 * sizeof(float)) +
         align256(bh * P * bwd_dw_floats(ks) * sizeof(float)) + align256(bh * P * sizeof(float)) +
         (bwd_split_differs(ks) ? 2 : 1) * wf + pad_bytes(d);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Chunks per workgroup of the standalone feature map: about 512 workgroups
// in all (each builds its frequency fragments once), at least one chunk each.
int fmap_chunks_per_wg(const flex_desc* d) {
  const long long total = (long long)nchunks_of(d) * d->B * d->H;
  long long c = total / 512;
  if (c < 1) c = 1;
  if (c > nchunks_of(d)) c = nchunks_of(d);
  return (int)c;
}

// Distillation-loss workspace: features of Q and K, z, per-query statistics,
// loss partials, dphi(Q), dphi(K) (io dtype), frequency-gradient and dtau
// partials.
struct AwdLayout {
  size_t phq, phk, z, stats, lpart, dphq, dphk, wpart, dtpart, total;
};
int awd_ntile(const flex_desc* d) { return (d->N + 63) / 64; }
AwdLayout awd_layout(const flex_desc* d) {
  const size_t bh = (size_t)d->B * d->H, N = (size_t)d->N, F = 2 * (size_t)d->m;
  const size_t io = d->io_dtype == FLEX_BF16 ? 2 : 4;
  const size_t nmat = d->variant == FLEX_NONSTATIONARY ? 2 : 1;
  const size_t parts = (size_t)flex::awd_parts(d->B, d->H, d->N);
  AwdLayout L;
  size_t off = 0;
  L.phq = off;    off += align256(bh * N * F * io);
  L.phk = off;    off += align256(bh * N * F * io);
  L.z = off;      off += align256(bh * F * sizeof(float));
  L.stats = off;  off += align256(bh * N * 2 * sizeof(float));
  L.lpart = off;  off += align256(bh * (size_t)awd_ntile(d) * sizeof(float));
  L.dphq = off;   off += align256(bh * N * F * io);
  L.dphk = off;   off += align256(bh * N * F * io);
  L.wpart = off;  off += align256((size_t)d->H * parts * nmat * d->m * d->d * sizeof(float));
  L.dtpart = off; off += align256((size_t)d->H * parts * sizeof(float));
  L.total = off;
  return L;
}
int32_t check_awd_desc(const flex_desc* d) {
  const int32_t st = check_desc_fields(d);
  if (st != FLEX_OK) return st;
  if (d->causal != 0) return FLEX_ERR_UNSUPPORTED;
  if (!flex::awd_shape_supported(d->io_dtype == FLEX_BF16, d->d, d->m)) return FLEX_ERR_UNSUPPORTED;
  return FLEX_OK;
}

}  // namespace

namespace flex {

namespace {
struct Timing {
  std::mutex mu;
  int kernel = 0;
  std::vector<hipEvent_t> ev;   // pairs (begin, end)
  size_t used = 0;              // completed pairs
  bool open = false;
  bool failed = false;
};
Timing& timing() {
  static Timing t;
  return t;
}
}  // namespace

void timing_mark(int kernel_class, hipStream_t st, bool begin) {
  Timing& t = timing();
  if (__atomic_load_n(&t.kernel, __ATOMIC_RELAXED) != kernel_class) return;
  std::lock_guard<std::mutex> lk(t.mu);
  if (t.kernel != kernel_class) return;
  if (begin) {
    if (2 * t.used + 2 > t.ev.size()) {
      hipEvent_t a, b;
      // timing-only events: no system-scope fence (cache writeback and
      // invalidation) when they are recorded, which would otherwise stall
      // the kernel that follows for several microseconds
      if (hipEventCreateWithFlags(&a, hipEventDisableSystemFence) != hipSuccess ||
          hipEventCreateWithFlags(&b, hipEventDisableSystemFence) != hipSuccess) { t.failed = true; return; }
      t.ev.push_back(a);
      t.ev.push_back(b);
    }
    if (hipEventRecord(t.ev[2 * t.used], st) != hipSuccess) t.failed = true;
    t.open = true;
  } else if (t.open) {
    if (hipEventRecord(t.ev[2 * t.used + 1], st) != hipSuccess) t.failed = true;
    t.open = false;
    ++t.used;
  }
}

}  // namespace flex

// Workspace of flex_linattn_fwd_noalloc: a file-scope device array.  Each GPU
// the library runs on holds its own copy at its own address until the process
// ends.  In host code `scratch` names a host-side stand-in, not device memory,
// so it is never passed to a kernel: its device address is looked up once per
// device (hipGetSymbolAddress, with that device current) and kept in a table.
static __device__ __align__(256) unsigned char scratch[FLEX_NOALLOC_SCRATCH_BYTES];

namespace {

// Validation of the forward's arguments (everything but the workspace).
int32_t check_fwd_args(const flex_desc* desc, const void* Q, const void* K, const void* V,
                       const float* W1, const float* W2, const float* tau, const void* O,
                       const float* den) {
  const int32_t st = check_desc(desc);
  if (st != FLEX_OK) return st;
  if (!Q || !K || !V || !W1 || !tau || !O) return FLEX_ERR_INVALID_ARG;
  if ((desc->variant == FLEX_NONSTATIONARY) != (W2 != nullptr)) return FLEX_ERR_INVALID_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(W1) || (W2 && !aligned16(W2)) ||
      !aligned16(O) || (den && !aligned16(den)))
    return FLEX_ERR_INVALID_ARG;
  return FLEX_OK;
}

// The forward on validated arguments with a workspace of at least
// ws_bytes_of(desc, FLEX_PASS_FWD) bytes at `base`.
int32_t run_fwd(const flex_desc* desc, const void* Q, const void* K, const void* V, const float* W1,
                const float* W2, const float* tau, void* O, float* den, char* base, hipStream_t stream,
                float* state_out = nullptr, int state_dv = 0) {
  FwdArgs a;
  memset(&a, 0, sizeof(a));
  a.Q = Q; a.K = K; a.V = V; a.tau = tau; a.O = O; a.den = den;
  a.state_out = state_out;
  a.state_m = desc->m;
  a.state_dv = state_dv > 0 ? state_dv : desc->dv;
  const Groups G = groups_of(desc);
  const KernelShape ks = attn_shape(desc);
  const size_t sb = fwd_group_state_bytes(desc);
  a.wfrag = base + G.n * sb;
  if (G.n > 1) {
    char* acc = base + G.n * sb + align256(wfrag_bytes(ks, desc->H));
    a.acc_num = reinterpret_cast<float*>(acc);
    a.acc_den = reinterpret_cast<float*>(acc + align256((size_t)desc->B * desc->H * desc->N * desc->dv * sizeof(float)));
  }
  const int P0 = pick_segments(desc);
  a.BH = desc->B * desc->H; a.H = desc->H; a.N = desc->N;
  a.nchunks = nchunks_of(desc);
  a.segments = P0;
  a.chunks_per_seg = (a.nchunks + a.segments - 1) / a.segments;
  a.sub = fwd_sub_of(desc, P0);
  a.fold = fwd_fold_of(desc, P0);
  a.pre_segs = pre_segs_of(desc, P0);
  if (desc->causal) {
    // the sweep's chunks of chunk_of(desc) tokens: a segment spans the same
    // tokens as its 64-token pre-pass chunks
    a.sweep_chunk = chunk_of(desc);
    a.sweep_groups = a.segments;
    a.sweep_cps = a.chunks_per_seg * (kChunk / a.sweep_chunk);
  } else {
    // chunks per non-causal sweep workgroup: up to kSweepChunks (or
    // kReadoutChunks), fewer when that leaves the CUs short of workgroups
    // (one, or for the token-split readout two, resident per CU)
    const int per_wg = readout_split(desc) ? 2 : 1;
    const int cap = readout_split(desc) ? kReadoutChunks : kSweepChunks;
    const long long per_cu = ((long long)a.nchunks * a.BH + per_wg * kCUs - 1) / (per_wg * kCUs);
    a.sweep_chunk = kChunk;
    a.sweep_cps = (int)(per_cu < 1 ? 1 : (per_cu > cap ? cap : per_cu));
    if (a.sweep_cps > a.nchunks) a.sweep_cps = a.nchunks;
    a.sweep_groups = (a.nchunks + a.sweep_cps - 1) / a.sweep_cps;
  }
  a.s_const = s_const_of(desc);
  const PadRows pr = pad_rows_of(desc, base + ws_bytes_of(desc, FLEX_PASS_FWD));
  for (int g = 0; g < G.n; ++g) {
    if (!group_rows(desc, G, pr, g, W1, W2, stream, &a.W1, &a.W2, &a.w_stride, &a.fvalid)) return FLEX_ERR_HIP;
    a.state = reinterpret_cast<float*>(base + g * sb);
    a.state_f0 = group_off(G, g);
    a.acc = G.n == 1 ? 0 : (g == 0 ? 1 : 2);
    const hipError_t e = launch_fwd(a, ks, false, stream);
    if (e != hipSuccess) return FLEX_ERR_HIP;
  }
  if (G.n > 1 && launch_fwd_finish(a, ks.bf16, desc->dv, stream) != hipSuccess) return FLEX_ERR_HIP;
  return FLEX_OK;
}

// The forward of a dv != d descriptor: run_fwd at the padded width on
// zero-padded copies in the workspace (padded_desc).
int32_t run_fwd_padded(const flex_desc* desc, const void* Q, const void* K, const void* V, const float* W1,
                       const float* W2, const float* tau, void* O, float* den, char* base, hipStream_t stream,
                       float* state_out = nullptr) {
  const flex_desc pd = padded_desc(desc);
  const ValuePad L = value_pad_of(desc, FLEX_PASS_FWD);
  char* vp = base + ws_bytes_of(&pd, FLEX_PASS_FWD);
  const size_t rows = (size_t)desc->B * desc->H * desc->N, hm = (size_t)desc->H * desc->m;
  const int io = desc->io_dtype == FLEX_BF16 ? 2 : 4, w = pd.d;
  if (desc->dv > desc->d) {
    if (launch_copy_cols(Q, desc->d, vp + L.q, w, rows, io, stream) != hipSuccess ||
        launch_copy_cols(K, desc->d, vp + L.k, w, rows, io, stream) != hipSuccess ||
        launch_copy_cols(W1, desc->d, vp + L.w1, w, hm, 4, stream) != hipSuccess ||
        (W2 && launch_copy_cols(W2, desc->d, vp + L.w2, w, hm, 4, stream) != hipSuccess))
      return FLEX_ERR_HIP;
    return run_fwd(&pd, vp + L.q, vp + L.k, V, reinterpret_cast<const float*>(vp + L.w1),
                   W2 ? reinterpret_cast<const float*>(vp + L.w2) : nullptr, tau, O, den, base, stream, state_out,
                   desc->dv);
  }
  if (launch_copy_cols(V, desc->dv, vp + L.v, w, rows, io, stream) != hipSuccess) return FLEX_ERR_HIP;
  // a prefill state keeps the caller's dv columns (the others are the zero padding)
  const int32_t r = run_fwd(&pd, Q, K, vp + L.v, W1, W2, tau, vp + L.o, den, base, stream, state_out, desc->dv);
  if (r != FLEX_OK) return r;
  return launch_copy_cols(vp + L.o, w, O, desc->dv, rows, io, stream) == hipSuccess ? FLEX_OK : FLEX_ERR_HIP;
}

constexpr int kMaxDevices = 64;
struct ScratchTable {
  std::mutex mu;
  void* ptr[kMaxDevices] = {};
};
ScratchTable& scratch_table() {
  static ScratchTable t;
  return t;
}

int32_t scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return FLEX_ERR_HIP;
  ScratchTable& t = scratch_table();
  std::lock_guard<std::mutex> lk(t.mu);
  if (!t.ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FLEX_ERR_HIP;
    t.ptr[dev] = p;
  }
  *out = t.ptr[dev];
  return FLEX_OK;
}

// The backward on validated arguments with a workspace of at least
// ws_bytes_of(desc, FLEX_PASS_BWD) bytes at `base`.
int32_t run_bwd(const flex_desc* desc, const void* Q, const void* K, const void* V, const float* W1,
                const float* W2, const float* tau, const void* O, const float* den, const void* dO, float* dQ,
                float* dK, float* dV, float* dW1, float* dW2, float* dtau, const void* fwd_ws, char* base,
                hipStream_t stream) {
  const KernelShape ks = attn_shape(desc);
  const Groups G = groups_of(desc);
  BwdArgs a;
  memset(&a, 0, sizeof(a));
  a.Q = Q; a.K = K; a.V = V; a.tau = tau; a.O = O; a.den = den; a.dO = dO;
  a.dQ = dQ; a.dK = dK; a.dV = dV;
  a.dtau = dtau;
  a.BH = desc->B * desc->H; a.B = desc->B; a.H = desc->H; a.N = desc->N;
  // the backward sweeps use BWD_CHUNK-token chunks over the forward's segments
  a.nchunks = (desc->N + BWD_CHUNK - 1) / BWD_CHUNK;
  a.segments = pick_segments(desc);
  {
    const int fcps = (nchunks_of(desc) + a.segments - 1) / a.segments;   // forward chunks per segment
    a.chunks_per_seg = fcps * (kChunk / BWD_CHUNK);
  }
  if (fwd_ws) {
    a.fsub = fwd_sub_of(desc, a.segments);
    a.ffold = fwd_fold_of(desc, a.segments);
    // with the forward's key-side states the scan would handle R' alone: the
    // dK/dV sweep sums its suffix itself when it reads at most kRFoldMax states
    a.rfold = desc->causal && a.segments - 1 <= kRFoldMax ? 1 : 0;
  }
  a.s_const = s_const_of(desc);
  const size_t bh = (size_t)a.BH, P = (size_t)a.segments;
  const size_t sb = align256(bh * P * bwd_state_floats(ks) * sizeof(float));
  const size_t gb = align256(bh * (size_t)a.N * 2 * sizeof(float));
  a.sstate = reinterpret_cast<float*>(base);
  a.rstate = reinterpret_cast<float*>(base + sb);
  a.gstats = reinterpret_cast<float*>(base + 2 * sb);
  a.dwpart = reinterpret_cast<float*>(base + 2 * sb + gb);
  a.dtaupart = reinterpret_cast<float*>(base + 2 * sb + gb + align256(bh * P * bwd_dw_floats(ks) * sizeof(float)));
  a.wfrag = base + 2 * sb + gb + align256(bh * P * bwd_dw_floats(ks) * sizeof(float)) + align256(bh * P * sizeof(float));
  a.wfrag_kv = bwd_split_differs(ks) ? static_cast<char*>(a.wfrag) + align256(wfrag_bytes(ks, desc->H)) : a.wfrag;
  a.dw_stride = desc->m * desc->d;
  const PadRows pr = pad_rows_of(desc, base + ws_bytes_of(desc, FLEX_PASS_BWD));
  for (int g = 0; g < G.n; ++g) {
    if (!group_rows(desc, G, pr, g, W1, W2, stream, &a.W1, &a.W2, &a.w_stride, &a.fvalid))
      return FLEX_ERR_HIP;
    const size_t woff = (size_t)group_off(G, g) * desc->d;   // this group's frequency rows
    a.dW1 = dW1 + woff;
    a.dW2 = dW2 ? dW2 + woff : nullptr;
    a.acc = g > 0;
    if (fwd_ws)
      a.fstate = reinterpret_cast<const float*>(static_cast<const char*>(fwd_ws) + g * fwd_group_state_bytes(desc));
    const hipError_t e = launch_bwd(a, ks, stream);
    if (e != hipSuccess) return FLEX_ERR_HIP;
  }
  return FLEX_OK;
}

// The backward of a dv != d descriptor: run_bwd at the padded width on
// zero-padded copies in the workspace (padded_desc), then the caller's columns
// of the padded gradients.
int32_t run_bwd_padded(const flex_desc* desc, const void* Q, const void* K, const void* V, const float* W1,
                       const float* W2, const float* tau, const void* O, const float* den, const void* dO,
                       float* dQ, float* dK, float* dV, float* dW1, float* dW2, float* dtau, const void* fwd_ws,
                       char* base, hipStream_t stream) {
  const flex_desc pd = padded_desc(desc);
  const ValuePad L = value_pad_of(desc, FLEX_PASS_BWD);
  char* vp = base + ws_bytes_of(&pd, FLEX_PASS_BWD);
  const size_t rows = (size_t)desc->B * desc->H * desc->N, hm = (size_t)desc->H * desc->m;
  const int io = desc->io_dtype == FLEX_BF16 ? 2 : 4, w = pd.d, f = (int)sizeof(float);
  if (desc->dv > desc->d) {
    if (launch_copy_cols(Q, desc->d, vp + L.q, w, rows, io, stream) != hipSuccess ||
        launch_copy_cols(K, desc->d, vp + L.k, w, rows, io, stream) != hipSuccess ||
        launch_copy_cols(W1, desc->d, vp + L.w1, w, hm, f, stream) != hipSuccess ||
        (W2 && launch_copy_cols(W2, desc->d, vp + L.w2, w, hm, f, stream) != hipSuccess))
      return FLEX_ERR_HIP;
    float* dWp2 = W2 ? reinterpret_cast<float*>(vp + L.dw2) : nullptr;
    const int32_t r = run_bwd(&pd, vp + L.q, vp + L.k, V, reinterpret_cast<const float*>(vp + L.w1),
                              W2 ? reinterpret_cast<const float*>(vp + L.w2) : nullptr, tau, O, den, dO,
                              reinterpret_cast<float*>(vp + L.dq), reinterpret_cast<float*>(vp + L.dk), dV,
                              reinterpret_cast<float*>(vp + L.dw1), dWp2, dtau, fwd_ws, base, stream);
    if (r != FLEX_OK) return r;
    if (launch_copy_cols(vp + L.dq, w, dQ, desc->d, rows, f, stream) != hipSuccess ||
        launch_copy_cols(vp + L.dk, w, dK, desc->d, rows, f, stream) != hipSuccess ||
        launch_copy_cols(vp + L.dw1, w, dW1, desc->d, hm, f, stream) != hipSuccess ||
        (W2 && launch_copy_cols(dWp2, w, dW2, desc->d, hm, f, stream) != hipSuccess))
      return FLEX_ERR_HIP;
    return FLEX_OK;
  }
  if (launch_copy_cols(V, desc->dv, vp + L.v, w, rows, io, stream) != hipSuccess ||
      launch_copy_cols(O, desc->dv, vp + L.o, w, rows, io, stream) != hipSuccess ||
      launch_copy_cols(dO, desc->dv, vp + L.dO, w, rows, io, stream) != hipSuccess)
    return FLEX_ERR_HIP;
  const int32_t r = run_bwd(&pd, Q, K, vp + L.v, W1, W2, tau, vp + L.o, den, vp + L.dO, dQ, dK,
                            reinterpret_cast<float*>(vp + L.dv), dW1, dW2, dtau, fwd_ws, base, stream);
  if (r != FLEX_OK) return r;
  return launch_copy_cols(vp + L.dv, w, dV, desc->dv, rows, f, stream) == hipSuccess ? FLEX_OK : FLEX_ERR_HIP;
}

}  // namespace

extern "C" {

int32_t flex_abi_version(void) { return FLEX_ABI_VERSION; }

int32_t flex_timing_enable(int32_t kernel) {
  if (kernel < FLEX_KERNEL_NONE || kernel > FLEX_KERNEL_AWD_WGRAD) return FLEX_ERR_INVALID_ARG;
  Timing& t = timing();
  std::lock_guard<std::mutex> lk(t.mu);
  t.kernel = kernel;
  t.used = 0;
  t.open = false;
  t.failed = false;
  return FLEX_OK;
}

int32_t flex_awd_loss(const flex_desc* desc, const void* Q, const void* K, const float* W1,
                      const float* W2, const float* tau, float* loss, float* dW1, float* dW2,
                      float* dtau, void* ws, size_t ws_bytes, void* stream) {
  const int32_t st = check_awd_desc(desc);
  if (st != FLEX_OK) return st;
  const bool ns = desc->variant == FLEX_NONSTATIONARY;
  if (!Q || !K || !W1 || !tau || !loss) return FLEX_ERR_INVALID_ARG;
  if (ns != (W2 != nullptr)) return FLEX_ERR_INVALID_ARG;
  const bool grads = dW1 != nullptr;
  if (grads && ns && !dW2) return FLEX_ERR_INVALID_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(W1) || (W2 && !aligned16(W2)) || !aligned16(loss) ||
      (grads && (!aligned16(dW1) || (ns && !aligned16(dW2)))))
    return FLEX_ERR_INVALID_ARG;
  const AwdLayout L = awd_layout(desc);
  if (!ws || ws_bytes < L.total || !aligned16(ws)) return FLEX_ERR_WORKSPACE;
  char* base = static_cast<char*>(ws);
  const hipStream_t sm = (hipStream_t)stream;
  // the features of Q and K, written once by the feature-map kernel
  FwdArgs f;
  memset(&f, 0, sizeof(f));
  f.W1 = W1; f.W2 = W2; f.tau = tau;
  f.BH = desc->B * desc->H; f.H = desc->H; f.N = desc->N;
  f.nchunks = nchunks_of(desc); f.segments = 1; f.chunks_per_seg = fmap_chunks_per_wg(desc); f.sub = 1;
  f.sweep_groups = 1; f.sweep_cps = f.nchunks;
  f.s_const = s_const_of(desc);
  f.w_stride = desc->m * desc->d;
  f.fvalid = desc->m; f.state_m = desc->m; f.state_f0 = 0;   // all frequencies in one launch
  const KernelShape ks = kshape(desc);
  f.Q = Q; f.O = base + L.phq;   // both matrices in one launch
  f.K = K; f.O2 = base + L.phk;
  if (launch_fwd(f, ks, true, sm) != hipSuccess) return FLEX_ERR_HIP;
  AwdArgs a;
  memset(&a, 0, sizeof(a));
  a.Q = Q; a.K = K; a.W1 = W1; a.W2 = W2; a.tau = tau;
  a.phq = base + L.phq; a.phk = base + L.phk;
  a.z = reinterpret_cast<float*>(base + L.z);
  a.stats = reinterpret_cast<float*>(base + L.stats);
  a.lpart = reinterpret_cast<float*>(base + L.lpart);
  a.dphq = base + L.dphq;
  a.dphk = base + L.dphk;
  a.wpart = reinterpret_cast<float*>(base + L.wpart);
  a.dtpart = reinterpret_cast<float*>(base + L.dtpart);
  a.loss = loss;
  a.dW1 = grads ? dW1 : nullptr;
  a.dW2 = grads && ns ? dW2 : nullptr;
  a.dtau = grads ? dtau : nullptr;
  a.BH = desc->B * desc->H; a.B = desc->B; a.H = desc->H; a.N = desc->N;
  a.ntile = awd_ntile(desc);
  a.parts = awd_parts(desc->B, desc->H, desc->N);
  a.c1 = (float)(1.4426950408889634 / sqrt((double)desc->d));
  a.log2n = (float)log2((double)desc->N);
  a.inv_n = (float)(1.0 / (double)desc->N);
  a.s_const = s_const_of(desc);
  return launch_awd(a, ks, grads, sm) == hipSuccess ? FLEX_OK : FLEX_ERR_HIP;
}

int32_t flex_decode_step(const flex_desc* desc, const void* q, const void* k, const void* v,
                         const float* W1, const float* W2, const float* tau, float* state, void* o,
                         float* den, void* stream) {
  const int32_t st = check_desc_fields(desc);
  if (st != FLEX_OK) return st;
  if (!decode_supported(desc)) return FLEX_ERR_UNSUPPORTED;
  if (!q || !k || !v || !W1 || !tau || !state || !o) return FLEX_ERR_INVALID_ARG;
  if ((desc->variant == FLEX_NONSTATIONARY) != (W2 != nullptr)) return FLEX_ERR_INVALID_ARG;
  if (!aligned16(W1) || (W2 && !aligned16(W2)) || !aligned16(state) || !aligned16(q) || !aligned16(k) ||
      !aligned16(v) || !aligned16(o) || (den && !aligned16(den)))
    return FLEX_ERR_INVALID_ARG;
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  a.q = q; a.k = k; a.v = v; a.W1 = W1; a.W2 = W2; a.tau = tau; a.state = state; a.o = o; a.den = den;
  a.BH = desc->B * desc->H; a.H = desc->H; a.d = desc->d; a.dv = desc->dv; a.m = desc->m;
  a.s_const = s_const_of(desc);
  const hipError_t e = launch_decode(a, desc->io_dtype == FLEX_BF16, (hipStream_t)stream);
  return e == hipSuccess ? FLEX_OK : FLEX_ERR_HIP;
}

int32_t flex_timing_read(double* total_ms, int64_t* launches) {
  if (!total_ms || !launches) return FLEX_ERR_INVALID_ARG;
  Timing& t = timing();
  std::lock_guard<std::mutex> lk(t.mu);
  double sum = 0.0;
  bool ok = !t.failed;
  for (size_t i = 0; i < t.used && ok; ++i) {
    float ms = 0.f;
    ok = hipEventSynchronize(t.ev[2 * i + 1]) == hipSuccess &&
         hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]) == hipSuccess;
    sum += ms;
  }
  *total_ms = sum;
  *launches = (int64_t)t.used;
  t.used = 0;
  t.open = false;
  t.failed = false;
  return ok ? FLEX_OK : FLEX_ERR_HIP;
}

const char* flex_status_string(int32_t s) {
  switch (s) {
    case FLEX_OK: return "ok";
    case FLEX_ERR_INVALID_ARG: return "invalid argument";
    case FLEX_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case FLEX_ERR_WORKSPACE: return "workspace missing or too small";
    case FLEX_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t flex_workspace_size(const flex_desc* desc, int32_t pass, size_t* bytes) {
  if (bytes) *bytes = 0;
  if (!bytes) return FLEX_ERR_INVALID_ARG;
  if (pass < FLEX_PASS_FEATURE_MAP || pass > FLEX_PASS_AWD) return FLEX_ERR_INVALID_ARG;
  if (pass == FLEX_PASS_AWD) {
    const int32_t sa = check_awd_desc(desc);
    if (sa != FLEX_OK) return sa;
    *bytes = awd_layout(desc).total;
    return FLEX_OK;
  }
  const int32_t st = pass == FLEX_PASS_FEATURE_MAP ? check_fmap_desc(desc) : check_desc(desc);
  if (st != FLEX_OK) return st;
  *bytes = ws_bytes_of(desc, pass);
  return FLEX_OK;
}

int32_t flex_feature_map(const flex_desc* desc, const void* X, const float* W1, const float* W2,
                         const float* tau, void* Phi, void* ws, size_t ws_bytes, void* stream) {
  (void)ws; (void)ws_bytes;
  const int32_t st = check_fmap_desc(desc);
  if (st != FLEX_OK) return st;
  if (!X || !W1 || !tau || !Phi) return FLEX_ERR_INVALID_ARG;
  if ((desc->variant == FLEX_NONSTATIONARY) != (W2 != nullptr)) return FLEX_ERR_INVALID_ARG;
  if (!aligned16(X) || !aligned16(W1) || (W2 && !aligned16(W2)) || !aligned16(Phi))
    return FLEX_ERR_INVALID_ARG;
  FwdArgs a;
  memset(&a, 0, sizeof(a));
  a.Q = X; a.tau = tau; a.O = Phi;
  a.BH = desc->B * desc->H; a.H = desc->H; a.N = desc->N;
  a.nchunks = nchunks_of(desc); a.segments = 1; a.chunks_per_seg = fmap_chunks_per_wg(desc); a.sub = 1;
  a.sweep_groups = 1; a.sweep_cps = a.nchunks;
  a.s_const = s_const_of(desc);
  a.w_stride = desc->m * desc->d;
  a.state_m = desc->m;
  // slices of the kernel's frequency count; a last slice it does not fill reads
  // only its own rows of W and writes only their columns
  KernelShape ks = kshape(desc);
  ks.m = fmap_slice_m(desc);
  for (int f0 = 0; f0 < desc->m; f0 += ks.m) {
    a.W1 = W1 + (size_t)f0 * desc->d;
    a.W2 = W2 ? W2 + (size_t)f0 * desc->d : nullptr;
    a.state_f0 = f0;
    a.fvalid = desc->m - f0 < ks.m ? desc->m - f0 : ks.m;
    if (launch_fwd(a, ks, true, (hipStream_t)stream) != hipSuccess) return FLEX_ERR_HIP;
  }
  return FLEX_OK;
}

int32_t flex_linattn_fwd(const flex_desc* desc, const void* Q, const void* K, const void* V,
                         const float* W1, const float* W2, const float* tau, void* O, float* den,
                         void* ws, size_t ws_bytes, void* stream) {
  const int32_t st = check_fwd_args(desc, Q, K, V, W1, W2, tau, O, den);
  if (st != FLEX_OK) return st;
  const size_t need = ws_bytes_of(desc, FLEX_PASS_FWD);
  if (!ws || ws_bytes < need || !aligned16(ws)) return FLEX_ERR_WORKSPACE;
  if (desc->dv != desc->d)
    return run_fwd_padded(desc, Q, K, V, W1, W2, tau, O, den, static_cast<char*>(ws), (hipStream_t)stream);
  return run_fwd(desc, Q, K, V, W1, W2, tau, O, den, static_cast<char*>(ws), (hipStream_t)stream);
}

int32_t flex_linattn_prefill(const flex_desc* desc, const void* Q, const void* K, const void* V,
                             const float* W1, const float* W2, const float* tau, void* O, float* den,
                             float* state, void* ws, size_t ws_bytes, void* stream) {
  const int32_t st = check_fwd_args(desc, Q, K, V, W1, W2, tau, O, den);
  if (st != FLEX_OK) return st;
  if (desc->causal != 1) return FLEX_ERR_UNSUPPORTED;
  if (!state || !aligned16(state)) return FLEX_ERR_INVALID_ARG;
  const size_t need = ws_bytes_of(desc, FLEX_PASS_FWD);
  if (!ws || ws_bytes < need || !aligned16(ws)) return FLEX_ERR_WORKSPACE;
  if (desc->dv != desc->d)
    return run_fwd_padded(desc, Q, K, V, W1, W2, tau, O, den, static_cast<char*>(ws), (hipStream_t)stream, state);
  return run_fwd(desc, Q, K, V, W1, W2, tau, O, den, static_cast<char*>(ws), (hipStream_t)stream, state);
}

int32_t flex_linattn_fwd_noalloc(const flex_desc* desc, const void* Q, const void* K, const void* V,
                                 const float* W1, const float* W2, const float* tau, void* O,
                                 float* den, void* stream) {
  const int32_t st = check_fwd_args(desc, Q, K, V, W1, W2, tau, O, den);
  if (st != FLEX_OK) return st;
  if (ws_bytes_of(desc, FLEX_PASS_FWD) > (size_t)FLEX_NOALLOC_SCRATCH_BYTES) return FLEX_ERR_WORKSPACE;
  void* ws = nullptr;
  const int32_t sst = scratch_of_current_device(&ws);
  if (sst != FLEX_OK) return sst;
  // the forward writes every workspace byte it reads (segment states, their
  // scan, fragments, group sums, padded copies), so the scratch needs no clearing
  if (desc->dv != desc->d)
    return run_fwd_padded(desc, Q, K, V, W1, W2, tau, O, den, static_cast<char*>(ws), (hipStream_t)stream);
  return run_fwd(desc, Q, K, V, W1, W2, tau, O, den, static_cast<char*>(ws), (hipStream_t)stream);
}

int32_t flex_linattn_bwd(const flex_desc* desc, const void* Q, const void* K, const void* V,
                         const float* W1, const float* W2, const float* tau, const void* O,
                         const float* den, const void* dO, void* dQ, void* dK, void* dV, float* dW1,
                         float* dW2, float* dtau, const void* fwd_ws, size_t fwd_ws_bytes, void* ws,
                         size_t ws_bytes, void* stream) {
  const int32_t st = check_desc(desc);
  if (st != FLEX_OK) return st;
  const bool ns = desc->variant == FLEX_NONSTATIONARY;
  if (!Q || !K || !V || !W1 || !tau || !O || !den || !dO || !dQ || !dK || !dV || !dW1)
    return FLEX_ERR_INVALID_ARG;
  if (ns != (W2 != nullptr) || ns != (dW2 != nullptr)) return FLEX_ERR_INVALID_ARG;
  const void* ptrs[] = {Q, K, V, W1, O, den, dO, dQ, dK, dV, dW1};
  for (const void* p : ptrs)
    if (!aligned16(p)) return FLEX_ERR_INVALID_ARG;
  if ((W2 && !aligned16(W2)) || (dW2 && !aligned16(dW2))) return FLEX_ERR_INVALID_ARG;
  const size_t need = ws_bytes_of(desc, FLEX_PASS_BWD);
  if (!ws || ws_bytes < need || !aligned16(ws)) return FLEX_ERR_WORKSPACE;
  if (fwd_ws && (fwd_ws_bytes < ws_bytes_of(desc, FLEX_PASS_FWD) || !aligned16(fwd_ws)))
    return FLEX_ERR_WORKSPACE;
  if (desc->dv != desc->d)
    return run_bwd_padded(desc, Q, K, V, W1, W2, tau, O, den, dO, static_cast<float*>(dQ), static_cast<float*>(dK),
                          static_cast<float*>(dV), dW1, dW2, dtau, fwd_ws, static_cast<char*>(ws),
                          (hipStream_t)stream);
  return run_bwd(desc, Q, K, V, W1, W2, tau, O, den, dO, static_cast<float*>(dQ), static_cast<float*>(dK),
                 static_cast<float*>(dV), dW1, dW2, dtau, fwd_ws, static_cast<char*>(ws), (hipStream_t)stream);
}

}  // extern "C"
