// Internal interface between the C ABI (flex_api.hip) and the kernel files.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>

namespace flex {

// Chunk length (tokens) of the backward sweeps; the forward uses 64, and a
// backward segment spans the same tokens as the forward segment (twice as many
// chunks).
constexpr int BWD_CHUNK = 32;

struct KernelShape {
  bool bf16;
  bool nonstationary;
  bool causal;
  int d, m;
};

struct FwdArgs {
  const void* Q;      // also the input X of the feature map
  const void* K;
  const void* V;
  const float* W1;
  const float* W2;
  const float* tau;
  void* O;            // also the output Phi of the feature map
  float* den;
  float* state;       // [BH][segments * sub][state floats]
  void* wfrag;        // per-head frequency fragments (prepared by k_prep_freqs)
  int BH, H, N;
  int nchunks, segments, chunks_per_seg;
  int sub;            // state pre-pass workgroups per segment (chunks_per_seg % sub == 0)
  int pre_segs;       // segments whose local state the pre-pass forms: all (non-causal),
                      // all but the last (causal: only exclusive prefixes are read)
  int fold;           // causal: 1 = no scan launch, each sweep workgroup sums its carry-in
                      // from the local states of the segments before its own (in the
                      // scan's order); 0 = the scan writes the carry-ins over each
                      // segment's first slot
  int sweep_groups;   // sweep workgroups per (b,h): the segments (causal) or chunk groups (non-causal)
  int sweep_cps;      // chunks per sweep workgroup
  int sweep_chunk;    // tokens per chunk of the causal sweep: 16, 32 or 64 (the
                      // pre-pass, the segments and the non-causal sweep use 64)
  float s_const;      // sigma/sqrt(m) or sigma/(2 sqrt(m))
  // Frequency groups: W1/W2 point at this group's rows, w_stride is the
  // element stride between heads.  acc = 0 writes O (and den) directly; 1 and
  // 2 write / add the group's numerator and denominator into acc_num
  // [BH][N][dv] and acc_den [BH][N] (fp32), which k_fwd_finish divides.
  // fvalid: rows of this group that are frequencies (the rest of the group's
  // rows are zero padding whose features the kernels mask to zero).
  int w_stride;
  int acc;
  int fvalid;
  float* acc_num;
  float* acc_den;
  // feature map of a second input in the same launch (grid.z = 2): X = K,
  // Phi = O2; nullptr K maps Q only
  void* O2;
  // causal prefill: the final state sum_j phi(K_j) [V_j ; 1]^T of every slice in
  // the decode layout (per slice S [2m][state_dv] row-major, then z [2m]);
  // state_f0 is the first frequency of this launch's group, state_m the total
  // m, state_dv the caller's value width (at most the kernel's: the columns
  // past it are the zero padding of a dv < d call).  NULL: none.
  float* state_out;
  int state_f0, state_m, state_dv;
};

struct BwdArgs {
  const void* Q;
  const void* K;
  const void* V;
  const float* W1;
  const float* W2;
  const float* tau;
  const void* O;
  const float* den;
  const void* dO;
  float* dQ;
  float* dK;
  float* dV;
  float* dW1;
  float* dW2;
  float* dtau;
  float* sstate;      // [BH][segments][state floats]: key-side prefix states
  float* rstate;      // [BH][segments][state floats]: query-side suffix states
  float* gstats;      // [BH][N][2]: 1/den_i and delta_i = dO_i . O_i
  float* dwpart;      // [2 sides][BH][segments][rows][d] frequency-gradient partials: the
                      // query side's in tile-major order (the dK/dV sweep starts from
                      // it), the key side's holding both sides' sums in [matrix][m][d]
  float* dtaupart;    // [BH][segments] partial dtau
  void* wfrag;        // per-head frequency fragments (prepared by k_prep_freqs)
  void* wfrag_kv;     // fragments of the dK/dV sweep (== wfrag when its split is the same)
  const float* fstate; // forward segment states ([BH][segments*fsub][state]) or NULL
  int fsub;           // forward pre-pass workgroups per segment
  int ffold;          // 1: fstate holds the local states (the forward ran no scan) and
                      // the dQ sweep sums its carry-in from them; 0: the carry-in of
                      // segment p is in slot p*fsub
  int rfold;          // causal with fstate: 1 = no scan launch, the dK/dV sweep sums its
                      // R' carry-in from the local states of the later segments (in the
                      // scan's order); 0 = the scan writes the suffixes over them
  int BH, B, H, N;
  int nchunks, segments, chunks_per_seg;
  float s_const;
  // Frequency groups: W1/W2 and dW1/dW2 point at this group's rows, w_stride
  // is the element stride between heads; acc = 1 adds dQ, dK, dV and dtau to
  // the outputs (a later group), 0 writes them.  fvalid: as in FwdArgs; the
  // reduce writes dW1/dW2 rows below it only, dw_stride elements apart per
  // head (W1/W2 of a padded group are a copy with a stride of their own).
  int w_stride;
  int acc;
  int fvalid;
  int dw_stride;
};

// Event bracketing of one kernel class (see flex_timing_enable); no-ops unless
// that class is selected.
void timing_mark(int kernel_class, hipStream_t st, bool begin);
enum KernelClass { KC_FWD_STATE = 1, KC_FWD_SWEEP = 2, KC_SCAN = 3, KC_BWD_PREPASS = 4,
                   KC_BWD_DQ = 5, KC_BWD_DKV = 6, KC_BWD_REDUCE = 7, KC_FEATURE_MAP = 8,
                   KC_DECODE = 9, KC_AWD_FWD = 10, KC_AWD_BWD_K = 11, KC_AWD_WGRAD = 12 };

// One decode step: one new token per (b,h) slice against a caller-owned state.
struct DecodeArgs {
  const void* q;      // [BH][d] io dtype
  const void* k;      // [BH][d]
  const void* v;      // [BH][dv]
  const float* W1;    // [H][m][d]
  const float* W2;    // [H][m][d] or NULL (stationary)
  const float* tau;   // [H]
  float* state;       // per slice S [2m][dv] then z [2m], fp32, updated in place
  void* o;            // [BH][dv] io dtype
  float* den;         // [BH] or NULL
  int BH, H, d, dv, m;
  float s_const;
};
size_t decode_smem_bytes(int d, int dv, int m);
hipError_t launch_decode(const DecodeArgs& a, bool bf16, hipStream_t st);

// Attention-weight distillation loss and its kernel-parameter gradient.
struct AwdArgs {
  const void* Q;      // [BH][N][d] io dtype
  const void* K;      // [BH][N][d]
  const float* W1;    // [H][m][d]
  const float* W2;    // [H][m][d] or NULL (stationary)
  const float* tau;   // [H]
  const void* phq;    // [BH][N][2m] io dtype: phi(Q), written by the feature map
  const void* phk;    // [BH][N][2m]: phi(K)
  float* z;           // [BH][2m] column sums of phi(K)
  float* stats;       // [BH][N][2]: (lse2_i + log2 N, 1 / (N den_i)) per query
  float* lpart;       // [BH][ntile] loss partial per 64-query tile
  void* dphq;         // [BH][N][2m] io dtype: dL/dphi(Q)
  void* dphk;         // [BH][N][2m] io dtype: dL/dphi(K)
  float* wpart;       // [H][parts][nmat][m][d] frequency-gradient partials
  float* dtpart;      // [H][parts] dtau partials
  float* loss;        // [BH]
  float* dW1;         // [H][m][d] or NULL (loss only)
  float* dW2;         // [H][m][d] or NULL
  float* dtau;        // [H] or NULL
  int BH, B, H, N, ntile, parts;
  float c1;           // log2(e) / sqrt(d): scaled logits in base 2
  float log2n;        // log2(N)
  float inv_n;        // 1 / N
  float s_const;
};
int awd_parts(int B, int H, int N);
// Supported (d, m) of the distillation loss; the launch returns
// hipErrorInvalidValue for any other shape.
bool awd_shape_supported(bool bf16, int d, int m);
hipError_t launch_awd(const AwdArgs& a, const KernelShape& ks, bool grads, hipStream_t st);

// fp32 floats of one (b,h,segment) state block for a shape.
size_t fwd_state_floats(const KernelShape& ks);
size_t bwd_state_floats(const KernelShape& ks);
size_t bwd_dw_floats(const KernelShape& ks);
// bytes of the per-head frequency fragments for H heads
size_t wfrag_bytes(const KernelShape& ks, int H);
bool bwd_split_differs(const KernelShape& ks);
int fwd_state_waves(const KernelShape& ks);
// Waves per SIMD of the forward state pre-pass (its launch attribute): two,
// except at d = 128 nonstationary, whose wave holds more than half a SIMD's
// registers.
constexpr int state_waves_per_eu(int d, bool ns) { return (d <= 64 || !ns) ? 2 : 1; }
int fwd_state_wgs_per_cu(const KernelShape& ks);

// state (or NULL): [BH][P*sub][E]; writes the exclusive prefix (causal) into
// slot p*sub of every segment p, or the total (non-causal) into slot 0.
// state_rev (or NULL): [BH][P][E] (sub must then be 1), scanned in the same
// launch in reverse: the exclusive suffix (causal) into slot p, or the total
// into slot 0.
// nread: slots of `state` that hold local states (the rest are taken as zero
// and never read); state_rev is read in full.
hipError_t launch_state_scan(float* state, float* state_rev, int BH, int P, int sub, int E, bool causal,
                             hipStream_t st, int nread);
hipError_t launch_fwd(const FwdArgs& a, const KernelShape& ks, bool feature_map_only, hipStream_t st);
// O = acc_num / acc_den (io dtype), den = acc_den, after the last frequency group.
hipError_t launch_fwd_finish(const FwdArgs& a, bool bf16, int dv, hipStream_t st);
// dst[h][rows][d] = the first rows_valid rows of src[h] (src_stride elements
// apart per head), zero after them: the frequency rows of a padded group.
hipError_t launch_pad_rows(const float* src, float* dst, int H, int rows_valid, int rows, int d, int src_stride,
                           hipStream_t st);
// dst [rows][cols_dst] = src [rows][cols_src] with the columns past cols_src
// zero (cols_dst > cols_src) or cut off (cols_dst < cols_src); elements of
// elem_bytes, rows of a whole number of 16-byte units, 16-byte aligned.
hipError_t launch_copy_cols(const void* src, int cols_src, void* dst, int cols_dst, size_t rows, int elem_bytes,
                            hipStream_t st);
hipError_t launch_bwd(const BwdArgs& a, const KernelShape& ks, hipStream_t st);
// The dQ sweep of one shape (flex_bwd_dq.hip): grouped_acc adds into an
// earlier frequency group's dQ; wr also does the pre-pass's query-side work;
// masked takes the variant for a padded frequency group.
template <class T, int D, int FW, int NW, bool NS>
hipError_t launch_bwd_dq(const BwdArgs& a, bool causal, bool grouped_acc, bool wr, bool masked, hipStream_t st);

}  // namespace flex
