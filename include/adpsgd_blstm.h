/*
 * adpsgd_blstm.h -- C ABI of the MI355X (gfx950) learner-step library.
 *
 * One learner of H-ADPSGD (Zhang et al., "A Highly Efficient Distributed Deep
 * Learning System for Automatic Speech Recognition", arXiv 1907.05701)
 * repeats one SGD step of a bidirectional-LSTM acoustic model (Section 5.2):
 * the LSTM stack forward and back-propagation through time over fixed-length
 * chunks, a linear bottleneck, a softmax cross-entropy over context-dependent
 * states, then the super-learner gradient reduction (eq. 6) and the ADPSGD
 * local update, i.e. one column of eq. 7 (SGD plus 0.5/0.5 averaging with one
 * ring neighbour).
 *
 * Conventions shared by every call:
 *   - All pointers named theta/grad/x/y/dy/... are DEVICE pointers allocated by
 *     the caller; no call allocates device memory (the allocation-free head
 *     entry point works in a static device array of the library, held from
 *     the library's load on each device that runs it).  State carried
 *     between calls lives in the caller's act_ws (saved activations, the
 *     recurrence status flag).  Host-side, the library keeps a per-device
 *     side stream with its events (created on first use by an eager
 *     blstm_bwd that overlaps work, see there) and the bookkeeping of the
 *     optional timing hooks.  Workspace sizes come from
 *     blstm_workspace_bytes().
 *   - Every call only enqueues work on `stream` (no host synchronisation) and
 *     returns 0 on success or a negative BLSTM_E* code; blstm_last_error()
 *     then returns a message for the calling thread.  No C++ exception crosses
 *     the ABI.
 *   - Frame-major activation layout: element (t, b, j) of a [T][B][W] tensor
 *     is at (t*B + b)*W + j.
 *   - Parameters are one flat float32 vector in PyTorch nn.LSTM order: for
 *     layer l = 0..L-1, direction 0 (forward) then 1 (reverse): W_ih [4H][D_l],
 *     W_hh [4H][H], b_ih [4H], b_hh [4H] with gate row blocks i, f, g, o
 *     (D_0 = D, D_l = 2H above); then W_l [P][2H], b_l [P], W_s [K][P], b_s [K].
 *   - precision BLSTM_BF16: GEMM operands (weights and activations) are bf16,
 *     accumulation and the cell state are float32, master weights and
 *     gradients are float32.  precision BLSTM_FP32: everything is float32.
 *     Activation buffers (y_top, workspaces) hold the precision's element type.
 */
#ifndef ADPSGD_BLSTM_H
#define ADPSGD_BLSTM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { BLSTM_FP32 = 0, BLSTM_BF16 = 1 };

enum {
  BLSTM_OK = 0,
  BLSTM_EINVAL = -1,       /* null pointer, bad dims, bad argument */
  BLSTM_EUNSUPPORTED = -2, /* shape/alignment the kernels do not handle */
  BLSTM_EHIP = -3          /* a HIP launch or runtime call failed */
};

/* adpsgd_step flags */
enum {
  ADPSGD_ORDER_EQ7 = 1u,   /* new = 0.5*(theta + peer) - lr*g (eq. 7 as printed);
                              default: new = 0.5*((theta - lr*g) + peer) */
  ADPSGD_WRITE_PEER = 2u   /* also store the averaged weights into theta_peer
                              (both columns of the pairing in T_k change) */
};

/* L layers, D input features, H cells per direction, P bottleneck units,
 * K classes, T frames per chunk, B sequences; precision BLSTM_FP32/BF16.
 * The paper's model is L=6, D=260, H=512, P=256, K=32000, T=21. */
typedef struct blstm_dims {
  int32_t L, D, H, P, K, T, B, precision;
} blstm_dims;

/* Number of float32 parameters in the flat layout (Section 5.2's "over 43
 * million parameters": 43,154,944 for the paper's model), or BLSTM_EINVAL. */
int64_t blstm_param_count(const blstm_dims* dims);

/* Sizes in bytes of the caller-allocated buffers for these dims:
 *   act_ws   -- activations saved by blstm_fwd for blstm_bwd, plus the
 *               backward's scratch; owned by the caller, opaque layout except
 *               for its last 256 bytes (the recurrence status flag, see
 *               blstm_recurrence_ok).
 *   head_ws  -- scratch of softmax_ce_fwd_bwd (logits, partial sums).
 *   theta_lp -- the bf16 operand copy of theta (n * 2 bytes; 0 for FP32).
 *   y_top    -- blstm_fwd output [T][B][2H] in the precision's element type.
 * Any output pointer may be NULL.  Returns 0 or BLSTM_EINVAL/EUNSUPPORTED. */
int blstm_workspace_bytes(const blstm_dims* dims, size_t* act_ws, size_t* head_ws,
                          size_t* theta_lp, size_t* y_top);

/* theta_lp[i] = bf16 round-to-nearest-even of theta[i], for i < n (the flat
 * layout, unpadded).  BF16 only; a no-op returning 0 for FP32. */
int blstm_pack_params(const blstm_dims* dims, const float* theta, void* theta_lp,
                      hipStream_t stream);

/* Forward pass of the LSTM stack (Section 5.2; cell as PyTorch nn.LSTM, each
 * chunk starting from h = c = 0).
 *   theta    [n] float32;  theta_lp [n] bf16 (BF16; ignored for FP32)
 *   x        [T][B][D] float32 features
 *   act_ws   workspace, written (saved gate pre-activations, cell states, hidden states)
 *   y_top    [T][B][2H] output of the top layer, forward half first. */
int blstm_fwd(const blstm_dims* dims, const float* theta, const void* theta_lp,
              const float* x, void* act_ws, void* y_top, hipStream_t stream);

/* Bottleneck, softmax and frame cross-entropy with their backward
 * (Section 5.2; eqs. 1-2 and 4).  With s = W_s (W_l y + b_l) + b_s per frame:
 *   *loss   = loss_scale * sum over frames of (logsumexp(s) - s[label])
 *   dy_top  [T][B][2H] float32 = dloss/dy_top
 *   grad    the head slots (W_l, b_l, W_s, b_s) of the flat float32 gradient
 *           are overwritten; the LSTM slots are not touched.
 * labels [T][B] int32 in [0, K) (not checked: out-of-range labels give an
 * undefined loss).  loss_scale is 1/(B*T) for the mean frame loss.
 * loss is a device float. */
int softmax_ce_fwd_bwd(const blstm_dims* dims, const float* theta, const void* theta_lp,
                       const void* y_top, const int32_t* labels, float loss_scale,
                       float* loss, float* dy_top, float* grad, void* head_ws,
                       hipStream_t stream);

/* softmax_ce_fwd_bwd without a head_ws argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation).  The head workspace is a static device
 * array of HEAD_STATIC_SCRATCH_BYTES held by each device the library runs on
 * until the process ends; dims whose head workspace (blstm_workspace_bytes'
 * head_ws) exceeds it are rejected with BLSTM_EUNSUPPORTED.  Same arguments,
 * results and errors as softmax_ce_fwd_bwd otherwise.  The call allocates
 * nothing (its first call on a device looks the array's address up once).
 * Calls that overlap on one device share the array and race: serialise them
 * (one stream, or events). */
#define HEAD_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int softmax_ce_fwd_bwd_static(const blstm_dims* dims, const float* theta, const void* theta_lp,
                              const void* y_top, const int32_t* labels, float loss_scale,
                              float* loss, float* dy_top, float* grad, hipStream_t stream);

/* Back-propagation through time of the LSTM stack (Section 5.2 model; the
 * gradient g of eq. 4 for the LSTM parameters) given dy_top = dloss/dy_top.
 * Per layer, top-down: the gate-gradient recurrence in reverse time
 * (dh = dy + W_hh^T da of the next step, dc, da for gates i, f, g, o), then
 * dW_ih = sum_t da x^T, dW_hh = sum_t da h_prev^T, db = sum_t da and the
 * gradient reaching the layer below, dX = W_ih^T da.
 *   theta, theta_lp  as for blstm_fwd
 *   act_ws  from blstm_fwd with the same theta and dims (saved gate
 *           pre-activations, cell and hidden states); also used as scratch,
 *           so a second blstm_bwd needs a new blstm_fwd first
 *   y_top   [T][B][2H] in the precision's type, from that blstm_fwd
 *   dy_top  [T][B][2H] float32
 *   grad    [n] float32: the LSTM slots are overwritten (b_ih and b_hh
 *           receive the same bias gradient); head slots are not touched.
 * Returns 0, BLSTM_EINVAL (NULL pointer, bad dims) or BLSTM_EHIP (launch
 * failure).  When not under stream capture the call may also run work on an
 * internal stream of the current device (created once, default priority);
 * that work is joined into `stream` before the call returns, so stream order
 * holds as for any other call.  ADPSGD_BLSTM_OVERLAP=0 disables it. */
int blstm_bwd(const blstm_dims* dims, const float* theta, const void* theta_lp,
              void* act_ws, const void* y_top, const float* dy_top, float* grad,
              hipStream_t stream);

/* Whether every recurrent exchange wait of the persistent kernels completed
 * since the previous blstm_recurrence_ok on act_ws (or since act_ws was first
 * used): the flag is sticky, so one query after many steps (or after replays
 * of a captured graph) covers all of them.  The persistent kernels are plain
 * launches when the occupancy query shows the whole grid resident at once;
 * if other streams or processes occupy CUs, a wait gives up after its bound
 * instead of hanging and the results of that call are not valid.  The flag
 * lives in the last 256 bytes of act_ws (an int32 at offset act_ws_bytes -
 * 256, nonzero after a give-up, and an initialisation tag); the query reads
 * it, clears it, and returns BLSTM_OK or BLSTM_EHIP with a message.
 * Synchronises `stream`; not during stream capture.
 * ADPSGD_BLSTM_COOPERATIVE=1 makes every persistent launch cooperative
 * (guaranteed residency, about 15 us more per launch). */
int blstm_recurrence_ok(const blstm_dims* dims, const void* act_ws, hipStream_t stream);

/* Super-learner reduction (eq. 6): out = scale * sum_{r=0}^{R-1} grads[r],
 * summed left to right in float32.  grads is a HOST array of R device
 * pointers (1 <= R <= 16), each to n floats; out may equal grads[0]. */
int replica_grad_reduce(const float* const* grads, int32_t R, int64_t n, float scale,
                        float* out, hipStream_t stream);

/* ADPSGD local update, one column of eq. 7, fused with the reduction above.
 * g = scale * sum_r grads[r] (float32, left to right), t = lr*g, then
 *   default:          theta = ((theta - t) + theta_peer) * 0.5
 *   ADPSGD_ORDER_EQ7: theta = ((theta + theta_peer) * 0.5) - t
 * every operation a single float32 rounding, no fused multiply-add.
 * ADPSGD_WRITE_PEER also stores the result into theta_peer.  theta_lp, if
 * not NULL, receives the bf16 copy of the new theta (as blstm_pack_params).
 * R = 1 with scale = 1 is the plain update.  theta, theta_peer and theta_lp
 * must not alias each other or the gradients. */
int adpsgd_step(float* theta, float* theta_peer, const float* const* grads, int32_t R,
                float scale, int64_t n, float lr, uint32_t flags, void* theta_lp,
                hipStream_t stream);

/* Message describing the last failure on the calling thread ("" if none). */
const char* blstm_last_error(void);

/* Optional kernel timing.  After blstm_timing_begin(prefix), every library
 * kernel whose name starts with prefix ("" = all) is bracketed by HIP events
 * on the stream it is launched on; a run of consecutive launches of one
 * per-time-step kernel shares one event pair (counted as that many
 * launches).  blstm_timing_end() waits for those events, fills up to cap
 * entries (one per kernel name: launches and summed milliseconds), stores
 * the number of names in *count and stops recording.  Host-side bookkeeping
 * only; not thread-safe. */
typedef struct blstm_kernel_time {
  char name[48];
  int32_t launches;
  double total_ms;
} blstm_kernel_time;

int blstm_timing_begin(const char* prefix);
int blstm_timing_end(blstm_kernel_time* out, int32_t cap, int32_t* count);

#ifdef __cplusplus
}
#endif

#endif /* ADPSGD_BLSTM_H */
