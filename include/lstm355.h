/*
 * lstm355.h -- C ABI of liblstm355: the per-worker training step of a stacked
 * LSTM / LSTMP network (forward pass + back-propagation through time) on one
 * AMD Instinct MI355X (gfx950).
 *
 * The paper (Section 2, "Background") describes a data-parallel training step
 * as every worker running a forward and a backward pass over its own
 * mini-batch, after which the workers all-reduce the gradients.  This library
 * computes one worker's part for the LSTM layers of GNMT and BigLSTM
 * (Section 4, "Methodology"): outputs, input gradients and the weight
 * gradients that would enter the all-reduce.  It performs no all-reduce and
 * no weight update.
 *
 * Cell (textbook LSTM without peepholes; gate blocks ordered i, f, g, o):
 *   z_t = W x_t + R h_{t-1} + b ;  i,f,o = sigmoid, g = tanh
 *   c_t = f*c_{t-1} + i*g ;  m_t = o*tanh(c_t) ;  h_t = m_t  or  P m_t (LSTMP)
 *
 * Conventions for every call below
 *   - All tensor pointers are DEVICE pointers, row-major, time-major:
 *     x[T][B][I] (row stride ldx), y[T][B][Ho] (row stride ldy), h0/hT[B][Hr],
 *     c0/cT[B][H], W[4H][I], R[4H][Hr], b[4H], P[Hp][H].  Hr = Ho = Hp when a
 *     projection is used, else H.
 *   - "Activation" tensors (x, y, h0, hT, dy, dhT, dx, dh0) and weights
 *     (W, R, P) use the handle dtype (bf16 bit patterns or fp32).  Cell
 *     tensors (c0, cT, dcT, dc0), the bias and every weight gradient are fp32.
 *   - The caller owns every buffer.  The handle owns only its host-side
 *     descriptor and tiling choice.  Buffers must be 16-byte aligned.
 *   - Every call is asynchronous on `stream` (a hipStream_t, NULL for the
 *     default stream, passed as void * so that this header needs no HIP
 *     header) and returns a status; nothing throws or aborts across this
 *     boundary.  Arguments are validated on the host before anything is
 *     launched.
 *   - Calls on one handle that use the same workspace must be ordered (same
 *     stream); overlapping calls need distinct workspaces.
 *   - `reserve_bytes` / `workspace_bytes` give the sizes of the caller's
 *     reserve and workspace.  A call whose buffers are shorter than the sizes
 *     its query functions report returns LSTM_ERR_WORKSPACE before anything
 *     is launched (the device is not touched).
 */
#ifndef LSTM355_H
#define LSTM355_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lstm_handle *lstm_handle_t;

typedef enum {
    LSTM_OK = 0,
    LSTM_ERR_INVALID_ARG = 1,  /* bad size, NULL required pointer, misalignment */
    LSTM_ERR_UNSUPPORTED = 2,  /* shape has no kernel configuration on this device */
    LSTM_ERR_WORKSPACE = 3,    /* a reserve or workspace shorter than the call needs */
    LSTM_ERR_HIP = 4,          /* a HIP runtime call or kernel launch failed */
    LSTM_ERR_TIMEOUT = 5       /* a grid barrier's watchdog expired (see lstm_check) */
} lstm_status_t;

typedef enum {
    LSTM_F32 = 0,   /* fp32 storage and fp32 matrix-core arithmetic */
    LSTM_BF16 = 1   /* bf16 storage; fp32 accumulation, gates and cell state.  The
                       XCD-local kernels store two intermediates in fp16: the input
                       projection in lstm_forward when it spans more than 1024 rows
                       T*B and at least 192 tiles of 256x256, and the saved
                       activated gates for 33 to 256 batch rows. */
} lstm_dtype_t;

typedef struct {
    int T, B, I, H;   /* steps, mini-batch rows, input width, cells */
    int Hp;           /* 0: plain LSTM; > 0: LSTMP with P[Hp][H] */
    lstm_dtype_t dtype;
    int reverse;      /* 1: visit t = T-1 .. 0 (reverse direction of a bidirectional layer) */
    long ldx, ldy;    /* elements between consecutive (t,b) rows of x / dx and y / dy; 0 = dense */
} lstm_desc_t;

/* Validates the descriptor (I, H and Hp must be multiples of 8; ldx >= I and
 * ldy >= Ho, both multiples of 8) and creates a handle.  Does not touch the GPU. */
lstm_status_t lstm_create(const lstm_desc_t *desc, lstm_handle_t *out);

/* Bytes of `reserve`: written by lstm_forward, read by lstm_backward.  Holds
 * the activated gates [T][B][4H] and cell states [T][B][H] (fp32), for LSTMP
 * the pre-projection outputs m[T][B][H], and for the layers whose XCD-local
 * kernels save the activated gates in fp16 (bf16, plain LSTM, H in {256, 512,
 * 1024}, 33 to 256 batch rows) a further [T][B][4H] fp16 region.  Its
 * contents are the library's own, valid only for lstm_backward on the same
 * handle and device. */
size_t lstm_reserve_size(lstm_handle_t h);

/* Bytes of `workspace` (scratch for one call at a time: barrier counters,
 * the gate gradients dz[T][B][4H], transposed weight copies). */
size_t lstm_workspace_size(lstm_handle_t h);

/* Forward pass over all T steps.
 *   x   [T][B][I] (stride ldx); h0 [B][Hr], c0 [B][H]: NULL means zeros.
 *   W, R, b, P: parameters; P must be NULL iff Hp == 0.
 *   y   [T][B][Ho] (stride ldy): h_t of every step, stored at time index t.
 *   hT, cT: final state (state after the last visited step), may be NULL.
 *   reserve: lstm_reserve_size bytes, kept for lstm_backward. */
lstm_status_t lstm_forward(lstm_handle_t h,
                           const void *x, const void *h0, const float *c0,
                           const void *W, const void *R, const float *b, const void *P,
                           void *y, void *hT, float *cT,
                           void *reserve, size_t reserve_bytes,
                           void *workspace, size_t workspace_bytes, void *stream);

/* lstm_forward without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It calls no allocating routine: its
 * scratch (the sync words of the persistent recurrences: barrier counter,
 * abort word, per-XCD claim masks) lives in a 64 KiB array that the library
 * keeps on each GPU until the process ends.  Arguments and results are those
 * of lstm_forward.  Layers whose forward needs more scratch than that (the
 * stepwise recurrence of wide LSTMP layers, whose split products need
 * partial sums) return LSTM_ERR_WORKSPACE with the sizes in
 * lstm_last_error_detail.  Every call on one GPU shares its array, so calls
 * that overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller; each call clears what must start at zero. */
lstm_status_t lstm_forward_noalloc(lstm_handle_t h,
                                   const void *x, const void *h0, const float *c0,
                                   const void *W, const void *R, const float *b, const void *P,
                                   void *y, void *hT, float *cT,
                                   void *reserve, size_t reserve_bytes, void *stream);

/* Forward pass of a stack of L unidirectional LSTM layers run as one layer
 * wavefront: layer l+1 starts a time step as soon as layer l has produced
 * that step, so the layers advance together a few steps apart instead of one
 * after another.  This is the pipelining of layers over the sequence that
 * the paper uses for model parallelism of GNMT and BigLSTM (Section 2,
 * "Background"; Section 4, "Model Parallel Splitting"), here spread over the
 * XCDs of one GPU.  The result equals L calls of lstm_forward with
 * x_{l+1} = y_l (or y_l + x_l for a residual layer, see below), zero initial
 * states and no final states.
 *   h[l]: handles of the layers (bf16, Hp = 0, not reversed, equal T, B, H;
 *     layer l >= 1 has I = H and dense x and y).
 *   x: the stack's input, as for lstm_forward on h[0].
 *   W[l], R[l], b[l]: parameters of layer l.
 *   y[l]: output of layer l [T][B][H] (the input of layer l+1).
 *   residual: NULL, or per layer 0/1; residual[l] = 1 makes layer l's output
 *     y[l] + (its input), the residual connection of the GNMT encoder
 *     (Section 4, "Model Parallel Splitting"); that sum, the input of layer
 *     l+1 (or the stack's output for the top layer), goes to ysum[l]
 *     [T][B][H].  A residual layer needs an input as wide as its output.
 *     The sums are rounded to bf16 as lstm_add rounds them.
 *   reserve[l]: reserve of layer l (lstm_reserve_size(h[l]) bytes), for
 *     lstm_backward on h[l] exactly as after lstm_forward; reserve_bytes is
 *     the size of each of them.
 *   workspace: at least the largest lstm_workspace_size of the handles.
 * Runs when L is 2..4, H = 1024 and B <= 32 on an MI355X whose XCD-local
 * path is enabled; otherwise returns LSTM_ERR_UNSUPPORTED and the caller
 * runs the layers one by one with lstm_forward (which rewrites anything this
 * call may have written). */
lstm_status_t lstm_forward_stack(int L, const lstm_handle_t *h, const void *x,
                                 const void *const *W, const void *const *R, const float *const *b,
                                 void *const *y, const int *residual, void *const *ysum,
                                 void *const *reserve, size_t reserve_bytes,
                                 void *workspace, size_t workspace_bytes, void *stream);

/* Back-propagation through time for the loss
 *   L = sum_t <dy_t, y_t> + <dhT, h_final> + <dcT, c_final>,
 * summed over the batch.  Needs the forward's x, h0, c0 (the same values),
 * W, R, P, its output y and its reserve.
 *   dy [T][B][Ho] (stride ldy); dhT [B][Hr], dcT [B][H]: NULL means zeros.
 *   dx [T][B][I] (stride ldx), dh0 [B][Hr], dc0 [B][H]: NULL = not wanted.
 *   dW [4H][I], dR [4H][Hr], db [4H], dP [Hp][H]: fp32 weight gradients,
 *     required (dP only for LSTMP).
 *   accumulate: 0 overwrites the weight gradients, 1 adds to them (gradient
 *     accumulation over several mini-batches before an all-reduce, the delayed
 *     update the paper uses in Section 4, "Measuring Epoch Counts to
 *     Convergence"). */
lstm_status_t lstm_backward(lstm_handle_t h,
                            const void *dy, const void *dhT, const float *dcT,
                            const void *x, const void *h0, const float *c0,
                            const void *W, const void *R, const void *P,
                            const void *y, const void *reserve, size_t reserve_bytes,
                            void *dx, void *dh0, float *dc0,
                            float *dW, float *dR, float *db, float *dP,
                            int accumulate, void *workspace, size_t workspace_bytes, void *stream);

/* Backward pass of a stack run forward by lstm_forward_stack, as a layer
 * wavefront: layer l-1's BPTT step t starts as soon as layer l has produced
 * dz_{l,t} and its input gradient dx_{l,t} = dz_{l,t} W_l (the upstream
 * gradient of layer l-1), so the layers' BPTT runs a few steps apart instead
 * of one after another; the weight gradients follow per layer.  The result
 * equals lstm_backward on each layer from the top down, with dy of layer l-1
 * = dx of layer l, zero initial states and no gradient for the final states.
 *   h[l], W[l], R[l], y[l], residual, ysum[l], reserve[l], reserve_bytes: as
 *     given to lstm_forward_stack (every layer with I = H: the stack's input
 *     x has the layers' width).  A residual layer's upstream gradient also
 *     reaches its input unchanged: the input gradient of layer l is dz_l W_l
 *     plus the gradient of layer l's output.
 *   dy: gradient of the stack's output (y[L-1], or ysum[L-1] when the top
 *     layer is residual), [T][B][H].
 *   x: the stack's input (layer 0's input).
 *   dx: gradient of x [T][B][H], NULL when not wanted.
 *   dW[l], dR[l], db[l]: fp32 weight gradients of layer l; accumulate as for
 *     lstm_backward.
 *   workspace: lstm_backward_stack_workspace_size(L, h) bytes (per-layer dz
 *     and the gradients passed between layers); workspace_bytes is its size.
 * Runs when L is 2..4, T >= 2, H = 1024 and B <= 32 on an MI355X whose
 * XCD-local path is enabled; otherwise returns LSTM_ERR_UNSUPPORTED and the
 * caller runs lstm_backward layer by layer. */
lstm_status_t lstm_backward_stack(int L, const lstm_handle_t *h, const void *dy, const void *x,
                                  const void *const *W, const void *const *R, const void *const *y,
                                  const int *residual, const void *const *ysum,
                                  const void *const *reserve, size_t reserve_bytes, void *dx,
                                  float *const *dW, float *const *dR, float *const *db, int accumulate,
                                  void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes lstm_backward_stack needs for these layers; 0 when the
 * stack's shapes do not fit the backward layer wavefront. */
size_t lstm_backward_stack_workspace_size(int L, const lstm_handle_t *h);

/* Environment: LSTM355_XCD_LAUNCH=cooperative makes the persistent
 * recurrence kernels of the bf16 path wait, as cooperative launches, until
 * all their workgroups (one per CU) can be resident.  By default they are
 * plain dispatches, which saves about 11 us of queue synchronisation per
 * launch but relies on the device not running other kernels beside them;
 * if it does, their waits time out and lstm_check reports LSTM_ERR_TIMEOUT.
 * Use the cooperative launch when other streams (for example collectives
 * overlapping the backward pass) share the device. */

/* Synchronises `stream` and reports whether any kernel of the library gave up
 * at a grid barrier on the current device since the last check
 * (LSTM_ERR_TIMEOUT; the device-wide flag is then cleared).  Outputs of such a
 * call are undefined.  `workspace` (the one the checked calls used) may be
 * NULL, as after lstm_forward_noalloc: the flags are kept per device. */
lstm_status_t lstm_check(lstm_handle_t h, void *workspace, void *stream);

/* Frees the handle.  NULL is a no-op. */
lstm_status_t lstm_destroy(lstm_handle_t h);

/* Static string naming a status. */
const char *lstm_status_string(lstm_status_t s);

/* Human-readable detail of the last failing call on this host thread (which
 * argument was rejected, or which HIP call failed and why).  Never NULL. */
const char *lstm_last_error_detail(void);

/* Diagnostics: the tiling chosen for this handle on the current device.
 * out8 = {fwd workgroups, fwd cells per workgroup, fwd batch rows per tile,
 * fwd variant, bwd workgroups, bwd cells per workgroup, bwd batch rows per
 * tile, bwd variant}; a workgroup count of 0 means no tiling fits.  Variant
 * 1000 marks the XCD-local kernels (bf16, plain LSTM, H in {256, 512, 1024}:
 * each XCD owns ceil(B/8) batch rows, each workgroup H/32 cells). */
lstm_status_t lstm_describe_tiling(lstm_handle_t h, int *out8);

/* Elementwise out[i] = a[i] + b[i] for i < n, in fp32 arithmetic, rounded to
 * `dtype` (in-place allowed).  Used to compose stacks: residual connections
 * (output = y + x) and the input gradient of a bidirectional layer (sum of
 * both directions' dx). */
lstm_status_t lstm_add(lstm_dtype_t dtype, size_t n, const void *a, const void *b, void *out, void *stream);

/* --- kernel timing ----------------------------------------------------------
 * When enabled, every kernel the library launches is bracketed by two HIP
 * events on its own stream, and its algorithmic FLOPs and bytes are recorded
 * per kernel class.  lstm_profile_read waits for the recorded events and
 * returns per-class totals; lstm_profile_reset drops them. */
typedef struct {
    char name[32];
    int launches;
    double total_ms;      /* sum of launch durations */
    double flops;         /* algorithmic FLOPs, summed over launches */
    double bytes;         /* algorithmic HBM bytes, summed over launches */
} lstm_kernel_stat_t;

lstm_status_t lstm_profile_enable(int on);
lstm_status_t lstm_profile_reset(void);
/* Writes up to `cap` classes into `out`, sets *n to the number written. */
lstm_status_t lstm_profile_read(lstm_kernel_stat_t *out, int cap, int *n);

#ifdef __cplusplus
}
#endif
#endif /* LSTM355_H */
