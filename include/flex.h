/*
 * flex.h -- C ABI of the MI355X (gfx950) random-Fourier-feature linear
 * attention library (Flexformer, arXiv 2606.27748).
 *
 * Notation follows the paper.  For one (batch b, head h) slice:
 *   X in {Q, K}: N x d rows, V: N x dv rows, m frequencies per matrix, d' = 2m.
 *   Stationary variant (Flexformer_s, Sec. 3.2 first paragraph; feature map
 *   Eq.(phi_n) of Sec. 3.1):
 *       phi(x) = s e(x) [cos(W x) ; sin(W x)],           s = sigma / sqrt(m)
 *   Nonstationary variant (Flexformer_n, Sec. 3.2, Eq.(phi_non)), with
 *   W'1 = (W1 + W2)/2 and W'2 = (W1 - W2)/2:
 *       phi(x) = s e(x) [cos(W'1 x) cos(W'2 x) ; sin(W'1 x) cos(W'2 x)],
 *                                                       s = sigma / (2 sqrt(m))
 *   Norm factor (Sec. 3.2, learnable scale exp(tau)): e(x) = exp(||x||^2 / exp(tau_h)).
 *   Attention, Eq.(linear att) of Sec. 2.2:
 *       O_i = phi(Q_i)^T S / phi(Q_i)^T z,  S = sum_j phi(K_j) V_j^T,  z = sum_j phi(K_j)
 *   with the sums over all j (non-causal) or over j <= i (causal; the paper's
 *   autoregressive language model, Sec. 4.2, read with an inclusive mask).
 *   den_i = phi(Q_i)^T z (per row) is returned for the backward pass.  No clamp
 *   or epsilon is applied: den_i = 0 yields inf/NaN exactly as the definition.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library never
 *     allocates, frees or synchronizes.  Work is enqueued on `stream` (a
 *     hipStream_t; NULL = the default stream) and runs asynchronously.
 *   - Layouts are contiguous row-major: Q, K [B,H,N,d]; V, O, dO [B,H,N,dv];
 *     den [B,H,N]; W1, W2 [H,m,d] fp32 (one frequency matrix per head, as in the
 *     paper's parameter analysis, Appendix B); tau [H] fp32; Phi [B,H,N,2m] with
 *     features ordered [cos block | sin block] as printed in Eq.(phi_n)/(phi_non).
 *     The frequencies are always per head, so the descriptor has no head stride
 *     for W1/W2: a caller who shares one matrix across heads passes it H times
 *     (H*m*d floats); dW1/dW2 are then per head and the caller sums them.
 *   - Pointers must be 16-byte aligned.
 *   - The workspace `ws` is caller-owned device memory of at least
 *     flex_workspace_size() bytes for the same descriptor and pass; its contents
 *     on entry do not matter.
 *   - All arguments are validated before any device work is enqueued.  An
 *     invalid descriptor, a required NULL pointer, a W2 / variant mismatch or a
 *     too-small workspace returns an error code with no device work.  A failed
 *     kernel launch returns FLEX_ERR_HIP.  No C++ exception crosses the ABI.
 *   - Results are deterministic (bitwise identical from run to run).
 *   - Supported shapes: N >= 1 (a ragged last chunk is masked); d and dv
 *     each in {32, 64, 128} with io_dtype FLEX_BF16 and d = dv = 32 with
 *     FLEX_F32; m a multiple of 16 up to 256; chunk in {0, 16, 32, 64}.
 *     Others return FLEX_ERR_UNSUPPORTED.  Every supported shape has the
 *     forward and the backward.  dv != d runs at width max(d, dv) on
 *     zero-padded copies in the workspace (Q, K and W when dv > d; V, O and dO
 *     when dv < d), which leave the results unchanged.  (d, m) = (32, 64), (64, 64), (64, 128) (bf16) and (128, 64)
 *     run as one pass; every other shape runs as frequency groups (of 128 at
 *     bf16 d = 64 when 128 divides m, else of 64, the first one zero-padded
 *     when 64 does not divide m) whose sums are combined in a fixed order (the
 *     forward workspace then holds an fp32 numerator/denominator buffer).
 *     With FLEX_BF16 and m < 48 the gradients' relative error can exceed 2e-2:
 *     rounding the features to bf16 alone costs 1.5-2.3% at m = 16.
 *     flex_feature_map takes the same d and m (it runs in slices of 64, 128
 *     or 256 frequencies by d, the last one partly filled).
 *   - io_dtype FLEX_F32 computes every contraction in fp32 (MFMA f32);
 *     FLEX_BF16 reads bf16 inputs, projects with a two-term bf16 split of the
 *     frequencies and contracts bf16 features with fp32 accumulation (the
 *     backward's dX = dP W' takes the frequencies rounded once to bf16, like
 *     dP itself).
 */
#ifndef FLEX_H
#define FLEX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FLEX_ABI_VERSION 7

typedef enum {
  FLEX_OK = 0,
  FLEX_ERR_INVALID_ARG = 1,  /* NULL descriptor / pointer, bad sizes or enums   */
  FLEX_ERR_UNSUPPORTED = 2,  /* valid but not implemented (shape, dtype)        */
  FLEX_ERR_WORKSPACE = 3,    /* workspace NULL or smaller than required         */
  FLEX_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed      */
} flex_status;

typedef enum { FLEX_F32 = 0, FLEX_BF16 = 1 } flex_dtype;
typedef enum { FLEX_STATIONARY = 0, FLEX_NONSTATIONARY = 1 } flex_variant;
typedef enum { FLEX_PASS_FEATURE_MAP = 0, FLEX_PASS_FWD = 1, FLEX_PASS_BWD = 2,
               FLEX_PASS_AWD = 3 } flex_pass;

typedef struct {
  int32_t B, H, N;      /* batch, heads, sequence length                           */
  int32_t d, dv;        /* head dimension of Q/K and of V                          */
  int32_t m;            /* frequencies per matrix (the paper's n); d' = 2m          */
  int32_t variant;      /* flex_variant                                             */
  int32_t causal;       /* 0: all j; 1: j <= i                                      */
  int32_t chunk;        /* causal chunk length C in {16, 32, 64}; 0 selects 64.  The
                           causal forward forms tril(phi(Q_c) phi(K_c)^T)[V_c ; 1]
                           inside each C-token chunk and carries earlier tokens
                           in the running state; results agree across C up to
                           rounding.  The non-causal forward, the backward and
                           the segment split do not depend on it.               */
  int32_t segments;     /* sequence segments per (b,h); 0 selects a heuristic       */
  int32_t io_dtype;     /* flex_dtype of Q, K, V, O, dO and Phi                     */
  int32_t grad_dtype;   /* flex_dtype of dQ, dK, dV; only FLEX_F32 is supported     */
  float sigma;          /* square root of the total spectral measure; 1 by default  */
} flex_desc;

/* ABI version of the loaded library (FLEX_ABI_VERSION). */
int32_t flex_abi_version(void);

/* Static description of a status code; never NULL. */
const char* flex_status_string(int32_t status);

/* Bytes of workspace needed by `pass` (flex_pass) for this descriptor.
 * Writes *bytes and returns FLEX_OK, or an error code for an invalid or
 * unsupported descriptor (then *bytes is 0). */
int32_t flex_workspace_size(const flex_desc* desc, int32_t pass, size_t* bytes);

/* Feature map phi~(X) of Eq.(phi_n) (stationary) or Eq.(phi_non) (nonstationary)
 * times the norm factor exp(||x||^2/exp(tau)).
 *   X   [B,H,N,d]   io_dtype, input rows
 *   W1  [H,m,d]     fp32, frequencies (omega, or omega_1 for the nonstationary variant)
 *   W2  [H,m,d]     fp32, omega_2; must be NULL for the stationary variant
 *   tau [H]         fp32, log of the norm-factor scale
 *   Phi [B,H,N,2m]  io_dtype output, [cos | sin] feature blocks
 * `dv`, `causal`, `chunk`, `segments` and `grad_dtype` are ignored (any value
 * is accepted); the workspace may be NULL (flex_workspace_size gives 0). */
int32_t flex_feature_map(const flex_desc* desc, const void* X, const float* W1,
                         const float* W2, const float* tau, void* Phi,
                         void* ws, size_t ws_bytes, void* stream);

/* Forward attention, Eq.(linear att), non-causal or causal.
 *   Q, K [B,H,N,d], V [B,H,N,dv]   io_dtype
 *   W1, W2, tau                    as for flex_feature_map
 *   O    [B,H,N,dv]  io_dtype output
 *   den  [B,H,N]     fp32 output phi(Q_i)^T z_i, or NULL if not wanted
 * φ(Q) and φ(K) are formed on chip and never written to memory. */
int32_t flex_linattn_fwd(const flex_desc* desc, const void* Q, const void* K,
                         const void* V, const float* W1, const float* W2,
                         const float* tau, void* O, float* den,
                         void* ws, size_t ws_bytes, void* stream);

/* Causal prefill for autoregressive generation (the language model of
 * Sec. 4.2): flex_linattn_fwd on a causal prefix of N tokens (same O and den,
 * bitwise), which also writes the state of the whole prefix,
 *     S' = sum_{j<N} phi(K_j) [V_j ; 1]^T   (Eq.(linear att)),
 * in the layout of flex_decode_step.  Decode steps started from it continue
 * the sequence: after t steps with tokens N .. N+t-1, the step's output equals
 * row N+t-1 of flex_linattn_fwd's causal output on all N+t tokens.
 *   state  fp32, B*H*2m*(dv+1) floats, overwritten: per (b,h) slice S [2m][dv]
 *          row-major, then z [2m], feature rows in [cos | sin] order.
 *   ws     flex_workspace_size(desc, FLEX_PASS_FWD) bytes, as for the forward.
 * desc->causal must be 1 (FLEX_ERR_UNSUPPORTED otherwise); a NULL or
 * misaligned state returns FLEX_ERR_INVALID_ARG.  Shapes as flex_linattn_fwd. */
int32_t flex_linattn_prefill(const flex_desc* desc, const void* Q, const void* K,
                             const void* V, const float* W1, const float* W2,
                             const float* tau, void* O, float* den, float* state,
                             void* ws, size_t ws_bytes, void* stream);

/* Bytes of the static device scratch that serves flex_linattn_fwd_noalloc
 * as its workspace (one array per GPU). */
#define FLEX_NOALLOC_SCRATCH_BYTES (32u << 20)

/* flex_linattn_fwd for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments and results as flex_linattn_fwd (bitwise), without the
 * workspace: the library keeps the forward's workspace in a file-scope device
 * array of FLEX_NOALLOC_SCRATCH_BYTES on each GPU it runs on, held until the
 * process ends.  The call allocates and frees nothing (no hipMalloc, no
 * allocating library routine); its first call on a device looks up that
 * device's array.  The caller still owns Q, K, V, W1, W2, tau, O and den.
 *   - A descriptor whose forward workspace (flex_workspace_size with
 *     FLEX_PASS_FWD) exceeds FLEX_NOALLOC_SCRATCH_BYTES returns
 *     FLEX_ERR_WORKSPACE with no device work (e.g. d = 128, m = 256 at
 *     B = 2, H = 16, N = 8192).
 *   - `stream` must belong to the current device (hipGetDevice); the array of
 *     that device is used.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents (the forward overwrites all of it that it reads): calls
 *     whose executions overlap on one GPU (several streams, several threads)
 *     race and give wrong results.  Issue them on one stream.
 *   - The backward cannot reuse this forward's segment states: pass
 *     fwd_ws = NULL to flex_linattn_bwd. */
int32_t flex_linattn_fwd_noalloc(const flex_desc* desc, const void* Q, const void* K,
                                 const void* V, const float* W1, const float* W2,
                                 const float* tau, void* O, float* den, void* stream);

/* Backward of flex_linattn_fwd for an upstream gradient dO (the paper gives no
 * backward; it is the derivative of the forward above).
 *   Q, K, V, W1, W2, tau  the forward inputs
 *   O, den               the forward outputs (den must not be NULL)
 *   dO   [B,H,N,dv]       io_dtype, gradient of the loss with respect to O
 *   dQ, dK [B,H,N,d], dV [B,H,N,dv]   grad_dtype outputs (overwritten)
 *   dW1 [H,m,d] fp32 output (overwritten); dW2 [H,m,d] fp32 output, required for
 *   the nonstationary variant and NULL for the stationary one
 *   dtau [H] fp32 output or NULL (overwritten when given)
 *   fwd_ws, fwd_ws_bytes  optional (NULL, 0): the workspace of the
 *        flex_linattn_fwd call that produced O and den, with the same
 *        descriptor and inputs, unchanged since that call.  It holds the
 *        forward's key-side segment states sum_j phi(K_j) [V_j ; 1]^T; given
 *        it, the backward reads them instead of recomputing them.  A workspace
 *        that does not match the call gives wrong gradients (no check is
 *        possible); one smaller than flex_workspace_size(desc, FLEX_PASS_FWD)
 *        returns FLEX_ERR_WORKSPACE. */
int32_t flex_linattn_bwd(const flex_desc* desc, const void* Q, const void* K,
                         const void* V, const float* W1, const float* W2,
                         const float* tau, const void* O, const float* den,
                         const void* dO, void* dQ, void* dK, void* dV,
                         float* dW1, float* dW2, float* dtau,
                         const void* fwd_ws, size_t fwd_ws_bytes,
                         void* ws, size_t ws_bytes, void* stream);

/* Recurrent decode step (causal attention one token at a time, the
 * autoregressive language model of Sec. 4.2): for every (b,h) slice, with the
 * new token's q, k, v, the prefix state S' = [S | z] of Eq.(linear att) takes
 * the token and the query reads it out:
 *     S <- S + phi(k) v^T,  z <- z + phi(k),  O = (phi(q)^T S) / (phi(q)^T z)
 * (the token attends to itself, as in the inclusive causal forward).  After t
 * calls from a zero state, O equals row t of flex_linattn_fwd's causal output
 * for the same tokens.
 *   q, k [B,H,d], v [B,H,dv]   io_dtype, the new token of each slice
 *   W1, W2, tau               as for flex_feature_map
 *   state fp32, B*H*2m*(dv+1) floats, caller-owned, updated in place; per
 *                             (b,h) slice S [2m][dv] row-major, then z [2m];
 *                             feature rows in [cos | sin] order; all zero for
 *                             an empty prefix.  (S and z are kept apart so
 *                             that S rows are 16-byte aligned.)
 *   o [B,H,dv] io_dtype, den [B,H] fp32 or NULL
 * desc->N, causal, chunk and segments are ignored.  Shapes: d and dv
 * multiples of 4 up to 128, m up to 1024; others return FLEX_ERR_UNSUPPORTED.  The
 * projection and the features are computed in fp32.  No workspace. */
int32_t flex_decode_step(const flex_desc* desc, const void* q, const void* k,
                         const void* v, const float* W1, const float* W2,
                         const float* tau, float* state, void* o, float* den,
                         void* stream);

/* Attention-weight distillation loss (App. A.3; the loss Sec. 4.3 uses to
 * distil softmax attention into the learnable kernel) and its gradient with
 * respect to the kernel parameters.  For every (b,h) slice, with the softmax
 * target P_ij = exp(Q_i.K_j/sqrt(d)) / sum_l exp(Q_i.K_l/sqrt(d)) and the
 * kernel's weights A_ij = phi(Q_i)^T phi(K_j) (flex_feature_map's phi):
 *     loss[b,h] = -(1/N) sum_i sum_j P_ij log(A_ij / sum_l A_il)
 * evaluated as printed: no clamp or epsilon, so a non-positive A_ij / den_i
 * gives NaN (or inf) for its slice.  P is a constant (the paper trains only
 * the kernel parameters): the gradients are those of sum_{b,h} loss[b,h] with
 * respect to W1, W2 and tau; there is no dQ or dK.
 *   Q, K [B,H,N,d]   io_dtype
 *   W1, W2, tau      as for flex_feature_map
 *   loss [B,H] fp32  required
 *   dW1 [H,m,d] fp32 or NULL: NULL computes the loss only (dW2 and dtau are
 *                    then ignored); otherwise dW2 [H,m,d] is required for the
 *                    nonstationary variant, and dtau [H] is optional.  The
 *                    outputs are overwritten.
 *   ws               flex_workspace_size(desc, FLEX_PASS_AWD) bytes: the
 *                    features of Q and K, per-query statistics and the
 *                    gradient partials; nothing of size N x N.
 * desc->causal must be 0 (the loss sums over every key): 1 returns
 * FLEX_ERR_UNSUPPORTED; dv, chunk and segments are ignored.  Shapes:
 * bf16 (d, m) in {(32,64), (64,64), (64,128)} and fp32 (32,64).  Logits, the
 * log-sum-exp and the logarithms are fp32; A is accumulated in fp32 from
 * io_dtype features.  Deterministic. */
int32_t flex_awd_loss(const flex_desc* desc, const void* Q, const void* K,
                      const float* W1, const float* W2, const float* tau,
                      float* loss, float* dW1, float* dW2, float* dtau,
                      void* ws, size_t ws_bytes, void* stream);

/* ---- Kernel timing (profiling aid) --------------------------------------
 * Kernel classes of the library.  When timing is enabled for one class, every
 * launch of a kernel of that class is bracketed by two hipEvents recorded on
 * the launch stream; flex_timing_read() waits for the recorded events and
 * returns the summed elapsed time.  Timing is off by default and then costs
 * nothing.  The event objects are created on first use and kept for reuse. */
typedef enum {
  FLEX_KERNEL_NONE = 0,
  FLEX_KERNEL_FWD_STATE = 1,    /* forward segment-state pre-pass            */
  FLEX_KERNEL_FWD_SWEEP = 2,    /* forward chunk sweep / readout              */
  FLEX_KERNEL_SCAN = 3,         /* segment prefix / suffix scan               */
  FLEX_KERNEL_BWD_PREPASS = 4,  /* backward segment-state pre-pass            */
  FLEX_KERNEL_BWD_DQ = 5,       /* backward query-side sweep (dQ)             */
  FLEX_KERNEL_BWD_DKV = 6,      /* backward key-side sweep (dK, dV)           */
  FLEX_KERNEL_BWD_REDUCE = 7,   /* frequency / tau gradient reduction         */
  FLEX_KERNEL_FEATURE_MAP = 8,  /* standalone feature map                     */
  FLEX_KERNEL_DECODE = 9,       /* recurrent decode step                      */
  FLEX_KERNEL_AWD_FWD = 10,     /* distillation loss (and dphi(Q)) pass       */
  FLEX_KERNEL_AWD_BWD_K = 11,   /* distillation dphi(K) pass                  */
  FLEX_KERNEL_AWD_WGRAD = 12    /* distillation chain rule to dW', dtau       */
} flex_kernel;

/* Select the kernel class to time (FLEX_KERNEL_NONE disables) and discard
 * pending records.  Not to be changed while launches are in flight. */
int32_t flex_timing_enable(int32_t kernel);

/* Wait for the recorded events; *total_ms = summed kernel time and
 * *launches = number of timed launches since the last enable/read; then clear.
 * Returns FLEX_ERR_HIP if an event query fails. */
int32_t flex_timing_read(double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* FLEX_H */
