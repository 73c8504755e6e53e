// kernels.hpp -- host-side launch interface of the liblstm355 kernels
// (declarations shared by api.cpp and the .hip translation units).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lstm355 {

enum class DType { F32 = 0, BF16 = 1 };

inline size_t dsize(DType t) { return t == DType::BF16 ? 2 : 4; }

// Kernel classes for the timing hooks (profile.cpp).
enum KClass {
    K_GEMM_GX = 0,   // input projection X W^T + b
    K_REC_FWD,       // persistent forward recurrence
    K_REC_BWD,       // persistent BPTT recurrence
    K_GEMM_DX,       // dX = dZ W
    K_GEMM_DW,       // dW = dZ^T X
    K_GEMM_DR,       // dR = dZ^T H_prev
    K_GEMM_DP,       // dP = dH^T M
    K_SMALL,         // transposes, column sums, fills, adds
    K_GEMM_DWR,      // [dW | dR] = dZ^T [X | H_prev] as one product
    K_NCLASS
};
const char *kclass_name(int k);

// Timing hooks: bracket one launch with events when profiling is on.
struct ProfScope {
    ProfScope(int kclass, hipStream_t s, double flops, double bytes);
    ~ProfScope();
    int k;
    hipStream_t s;
    double flops, bytes;
    void *ev0;
};

// Work a launch can take on beside its own, spread over all of its
// workgroups once they have finished their own work (so that the extra
// stores do not delay the waits of its main loop): fill rows of 16-bit
// elements with a value, clear 32-bit words, and sum the rows of a small
// fp32 matrix into a vector (deterministic, in row order).  It saves the
// separate launches of these bandwidth-trivial steps.
struct SideJob {
    uint16_t *fill = nullptr;   // fill[r*fill_ld + c] = fill_v, r < fill_rows, c < fill_cols
    long fill_rows = 0;
    int fill_cols = 0;
    long fill_ld = 0;
    uint16_t fill_v = 0;
    unsigned *clr = nullptr;    // clr[i] = 0, i < clr_n
    int clr_n = 0;
    const float *sum_src = nullptr;   // sum_dst[c] (+)= sum_{r < sum_rows} sum_src[r*sum_cols + c]
    int sum_rows = 0, sum_cols = 0;
    float *sum_dst = nullptr;
    int sum_acc = 0;
};

// C[m][n] (beta ? C : 0) + sum_k A(m,k) B(n,k) (+ bias[n])
//   A(m,k) = a_kmajor ? A[m*lda + k] : A[k*lda + m]
//   B(n,k) = b_kmajor ? B[n*ldb + k] : B[k*ldb + n]
// Inputs share one element type; C is fp32 or the input type.
struct GemmDesc {
    DType in;
    bool out_f32;
    bool a_kmajor, b_kmajor;
    int M, N, K;
    const void *A; long lda;
    const void *B; long ldb;
    void *C; long ldc;
    const float *bias;
    int beta;
    float *splitk_ws;          // optional fp32 scratch for split-K partials
    size_t splitk_ws_floats;
    // Optional second column block (bf16, both operands m-major only): columns
    // n >= N1 of the product use B2 / B3 instead of B and are written to C2:
    //   C2[m][n-N1] (+)= sum over k of A(m,k) * S(n-N1, k), where row k of the
    //   operand S is B3 row (k - hlo) for k in [hlo, hlo+hlen) (skipped when
    //   B3 is NULL) and B2 row (k + yoff) for k in [ylo, yhi).
    // With B3, stages of 32 k never straddle those ranges (hlo, hlen, ylo,
    // yhi are multiples of 32).  Without B3 the second block runs over
    // [ylo, yhi) alone, from any ylo (rows of A past yhi read as zero).
    int N1 = 0;                // 0: no second block
    const void *B2 = nullptr; long ldb2 = 0; long b2_bytes = 0;
    const void *B3 = nullptr; long ldb3 = 0; long b3_bytes = 0;
    int ylo = 0, yhi = 0, yoff = 0, hlo = 0, hlen = 0;
    void *C2 = nullptr; long ldc2 = 0;
    SideJob side;              // done by the product's workgroups after their tiles
    // Optional fused LSTM cell update (bf16 operands, both k-major, fp32 C
    // accumulated into, N = 4 * cell_h): C holds the gate pre-activations of
    // H = cell_h cells in row blocks (i, f, g, o).  Instead of storing z, the
    // product stores the activations into C, c = f*cprev + i*g into cell_c,
    // m = o*tanh(c) (bf16) into cell_m[row*cell_ldm + j] and, if non-NULL,
    // c into cell_cT.  cell_prev NULL means a zero previous cell state.
    int cell_h = 0;
    const float *cell_prev = nullptr;
    float *cell_c = nullptr;
    void *cell_m = nullptr; long cell_ldm = 0;
    float *cell_cT = nullptr;
    // Batch: nbatch (<= 4) products of this shape in one launch, batch[i]
    // giving product i's A, B, B2, C, C2 and side-job sum pointers (the
    // other fields are this descriptor's).  One product follows another, so
    // the stores of one overlap the main loop of the next.  Never split
    // along K.
    int nbatch = 1;
    const GemmDesc *batch = nullptr;
    // Partials: the product split along K into exactly this many parts (> 1),
    // each part's fp32 sum written to splitk_ws[part][M][N] and left for the
    // caller to add up (no reduction runs; C, bias and beta are not used).
    int partials = 0;
    // fp16 C (bf16 operands, both k-contiguous, no accumulation into C): the
    // forward's input projection on the tiles gemm_f16_ok accepts.
    bool out_f16 = false;
};
// Whether `gemm` can run the fused cell update for descriptor d.
bool gemm_cell_ok(const GemmDesc &d);
// Whether `gemm` can run descriptor d with an fp16 C (out_f16).
bool gemm_f16_ok(const GemmDesc &d);
hipError_t gemm(const GemmDesc &d, hipStream_t s, int kclass);
// Whether a descriptor with a second column block (N1 > 0) can run.
bool gemm_dual_ok(const GemmDesc &d);

// Small kernels.
// dst[c][r] = src[r][c]; `side` (optional) is done by the same launch.
hipError_t transpose(DType t, const void *src, int rows, int cols, void *dst, hipStream_t s,
                     const SideJob *side = nullptr);
// Up to FILL_MAX word ranges, each filled with its own value: p[r][0..n[r]) = v[r].
constexpr int FILL_MAX = 16;
struct FillRanges {
    uint32_t *p[FILL_MAX];
    long n[FILL_MAX];
    uint32_t v[FILL_MAX];
    int count;
};
hipError_t fill_u32(void *p, size_t n, uint32_t v, hipStream_t s);
// p[r*ld + c] = v for r < rows, c < cols (16-bit elements).
hipError_t fill_rows_u16(void *p, long rows, int cols, long ld, uint16_t v, hipStream_t s);
// dst[c] (+)= sum_r src[r][c] over a [rows][cols] matrix of element type t, in fp32, deterministic;
// `partial` holds colsum_partial_floats(rows, cols) floats of scratch.
size_t colsum_partial_floats(int rows, int cols);
// dst[c] (+)= sum_{r < rows} src[r][c] for fp32 partial rows, in row order.
hipError_t sum_rows(const float *src, int rows, int cols, float *dst, int accumulate, hipStream_t s);
hipError_t colsum(DType t, const void *src, int rows, int cols, float *partial, float *dst, int accumulate, hipStream_t s);
hipError_t add(DType t, size_t n, const void *a, const void *b, void *out, hipStream_t s);
// dst[r*ldd + c] = src[r*lds + c] for r < rows, c < cols.
hipError_t copy_rows(DType t, long rows, int cols, const void *src, long lds, void *dst, long ldd, hipStream_t s);
// Cell update of one step for B rows x H cells (stepwise recurrence):
// gates_t [B][4H] holds the pre-activations on entry and the activations on
// exit; cprev [B][H] (NULL: zeros); writes c_t [B][H], m_out (storage type,
// row stride ldm), optionally h_copy (row stride ldh) and cT.
hipError_t gates_forward(DType t, int B, int H, float *gates_t, const float *cprev, float *c_t, void *m_out, long ldm,
                         void *h_copy, long ldh, float *cT, int kclass, hipStream_t s);
// Gate gradients of one step: the gradient of m_t is dm + dy + dh + dhT
// (each may be NULL); dcn [B][H] carries dc (read, then overwritten with the
// carry to the previous step); writes dz_t [B][4H] and, if given, dc0.
hipError_t gates_backward(DType t, int B, int H, const float *dm, const void *dy, long ldy, const float *dh,
                          const void *dhT, const float *gates_t, const float *c_t, const float *cprev, float *dcn,
                          void *dz_t, float *dc0, int kclass, hipStream_t s);

// Persistent recurrence kernels (recurrent.hip).
struct RecShape {
    int T, B, I, H, Hp, reverse;
    long ldy;
};
struct RecTiling {
    int HN;      // cells per workgroup
    int BM;      // batch rows per tile
    int nHT;     // hidden tiles
    int nBT;     // batch tiles
    int G;       // workgroups (cooperative grid)
    int bgroups; // workgroups per hidden tile
    int variant; // kernel instantiation index
    size_t lds;  // dynamic LDS bytes
};
// Chooses a tiling for the forward / backward kernels; false if none fits.
bool plan_forward(DType t, const RecShape &sh, int num_cus, RecTiling *out);
bool plan_backward(DType t, const RecShape &sh, int num_cus, RecTiling *out);

struct FwdBufs {
    const void *R, *P, *h0;
    const float *c0;
    float *gates;   // [T][B][4H]: in Gx (with bias), out activated gates
    float *cs;      // [T][B][H]
    void *ms;       // [T][B][H] (LSTMP)
    void *y;
    void *hT;
    float *cT;
    unsigned *sync;
    // Optional [T][B][4H] fp16 Gx (XCD-local forward only): the input
    // projection is read from here instead of from gates.
    const void *gx16 = nullptr;
    // Optional [T][B][4H] fp16 activated gates saved for the backward
    // (XCD-local forward only, xcd_act16 layers), instead of fp32 into gates.
    void *act16 = nullptr;
};
hipError_t launch_forward(DType t, const RecShape &sh, const RecTiling &tl, const FwdBufs &b, hipStream_t s);

struct BwdBufs {
    const void *Rt;     // R^T [Hr][4H]
    const void *Pt;     // P^T [H][Hp] (LSTMP)
    const void *dy;     // [T][B][Ho] stride ldy
    const void *dhT;
    const float *dcT;
    const void *h0;
    const float *c0;
    const float *gates, *cs;
    const void *act16;  // XCD-local backward of an xcd_act16 layer: the forward's fp16 activated gates
    void *dz;           // [T][B][4H]
    void *dH;           // [T][B][Hp] (LSTMP)
    float *dcn;         // [B][H] carry of dc between steps
    float *dhn;         // [B][H] carry of dh between steps (plain LSTM)
    void *dh0;
    float *dc0;
    float *dbpart;      // XCD-local kernel: [8][4H] per-XCD partial bias gradients
    unsigned *sync;
};
hipError_t launch_backward(DType t, const RecShape &sh, const RecTiling &tl, const BwdBufs &b, hipStream_t s);

// Workspace layout of the sync block (u32 words); the words a kernel uses are
// zeroed before it is launched.
constexpr size_t SYNC_BYTES = 4096;
constexpr int SYNC_COUNT0 = 0;     // barrier counter of the generic kernels
constexpr int SYNC_ABORT = 64;     // abort flag of the generic kernels
constexpr int SYNC_WORDS = 128;    // words cleared before a generic launch
constexpr int XCD_FLAGS = 256;     // words of the XCD-local kernels (257 words)
constexpr int XCD_CLAIM = 0;       // 8 per-XCD masks of claimed workgroup slots, relative to XCD_FLAGS
constexpr int XCD_ABORT = 256;     // abort flag, relative to XCD_FLAGS
constexpr int XCD_WORDS = 257;     // words cleared before an XCD-local launch

// Sticky error bits of the library (device variable): 1 = a watchdog expired,
// 2 = an XCD-local launch did not give every (XCD, slot) role exactly one workgroup.
constexpr unsigned TRIP_WATCHDOG = 1u, TRIP_PLACEMENT = 2u;

// XCD-local recurrences (recurrent_xcd.hip): bf16, plain LSTM, H in {256,
// 512, 1024}, exactly 256 CUs.
bool xcd_path_ok(DType t, const RecShape &sh, int num_cus);
constexpr int XCD_VARIANT = 1000;   // variant reported by lstm_describe_tiling for these kernels
void xcd_path_disable();
hipError_t xcd_tripped_read_and_clear(unsigned *tripped);   // like watchdog_read_and_clear
unsigned long long watchdog_ticks();
// The exchanged rows (y forward, dz backward) must hold XCD_NOT_READY and the
// XCD_WORDS words at XCD_FLAGS of the sync block must be zero when these
// kernels start: the launch functions prepare both unless `prepared` says an
// earlier launch on the stream (xcd_prep_forward / xcd_prep_backward as a
// side job) already did.
constexpr uint16_t XCD_NOT_READY = 0xffffu;
// Layer wavefront forward of a stack of L (2..4) unidirectional bf16 layers
// (H = 1024, at most 32 batch rows, zero initial states, y dense): with x
// NULL, layer 0's input projection must already be in ly[0].gates (with
// bias); with x given ([T][B][H], dense), the launch computes it.  Layers
// >= 1 take their input from the layer below.  Fills the exchanged rows and
// the flags itself.
struct WaveBufs {
    const void *R, *W;
    const float *bias;
    float *gates, *cs;
    void *y;
    // the layer below is residual: this layer's input is y of the layer below
    // plus in_b (written in the launch when poll_b), formed by this layer's
    // projection and stored into `sum`; NULL / 0 otherwise
    const void *in_b;
    void *sum;
    int poll_b;
};
bool wave_path_ok(const RecShape &sh, int num_cus);
hipError_t launch_forward_wave(const RecShape &sh, int L, const void *x, const WaveBufs *ly, unsigned *sync,
                               unsigned long long timeout, hipStream_t s);
// Backward of the layer wavefront (I = H = 1024 for every layer): Rt, Wt are
// R^T and W^T [H][4H] (Wt NULL: no input gradient for that layer); dz
// [T][B][4H] per layer; dy the upstream gradient (the stack's for the top
// layer, else the dx of the layer above, which this launch writes: dy_fill
// is the same buffer, armed before the launch); dbp [4H] the bias gradient.
struct WaveBwdBufs {
    const void *R, *W;   // R_l, W_l [4H][H] (W NULL: no input gradient wanted)
    const float *gates, *cs;
    void *dz;
    const void *dy;
    void *dy_fill;   // dy when the launch writes it (layers below the top), else NULL
    void *dx;
    float *dbp;
    int residual;    // the layer's output is y + its input: dx also receives dy (the identity path)
};
// The fills launch_backward_wave needs before its launch (flags, dz, the
// upstream gradients written inside the launch); with `prefilled` the caller
// has performed them.
FillRanges backward_wave_fills(const RecShape &sh, int L, const WaveBwdBufs *ly, unsigned *sync);
hipError_t launch_backward_wave(const RecShape &sh, int L, const WaveBwdBufs *ly, unsigned *sync,
                                unsigned long long timeout, hipStream_t s, bool prefilled = false);
SideJob xcd_prep_forward(const RecShape &sh, const FwdBufs &b);
// Whether the XCD-local kernels of a layer of this shape save the activated
// gates in fp16 (in their own reserve region) rather than fp32 into gates:
// layers with 5 to 32 batch rows per XCD, which the layer wavefront (at most
// 4 rows per XCD) never takes.  A fixed property of the layer, so that the
// forward and the backward agree on it.
bool xcd_act16(DType t, const RecShape &sh);
SideJob xcd_prep_backward(const RecShape &sh, const BwdBufs &b);
hipError_t launch_forward_xcd(const RecShape &sh, const FwdBufs &b, unsigned long long timeout, hipStream_t s,
                              bool prepared = false);
hipError_t launch_backward_xcd(const RecShape &sh, const BwdBufs &b, unsigned long long timeout, hipStream_t s,
                               bool prepared = false);

// Stepwise recurrences (stepwise.cpp): per step, the recurrent product runs
// on the matrix-core GEMM, followed by a pointwise cell kernel (and, for
// LSTMP, the projection product).  Used where the weights cannot stay
// resident in a persistent kernel.
constexpr int STEPWISE_VARIANT = 2000;   // variant reported by lstm_describe_tiling
struct StepwiseArgs {
    const void *R, *P;           // R [4H][Hr], P [Hp][H]
    float *splitk_ws;            // split-K partials of the per-step products
    size_t splitk_ws_floats;
};
hipError_t forward_stepwise(DType t, const RecShape &sh, const FwdBufs &b, const StepwiseArgs &w, hipStream_t s);
hipError_t backward_stepwise(DType t, const RecShape &sh, const BwdBufs &b, const StepwiseArgs &w, hipStream_t s);

// Reads (synchronously) and clears the library's sticky watchdog word on the
// current device: nonzero if a grid barrier gave up since the last call.
hipError_t watchdog_read_and_clear(unsigned *tripped);

}  // namespace lstm355
