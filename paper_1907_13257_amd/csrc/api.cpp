// api.cpp -- the C ABI of liblstm355: argument validation, buffer layout
// of `reserve` and `workspace`, and the order of kernel launches for one
// layer's forward pass and back-propagation through time.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>

#include "../../include/lstm355.h"
#include "kernels.hpp"

using namespace lstm355;

struct lstm_handle {
    lstm_desc_t d;
    DType dt;
    size_t es;
    int Hr;
    long ldx, ldy;
    long TB, G4;
    // reserve layout (bytes)
    size_t r_gates, r_cs, r_ms, r_act16, r_total;   // r_act16: 0 when the layer has no fp16 activations region
    // workspace layout (bytes)
    size_t w_sync, w_dz, w_rt, w_pt, w_dH, w_dcn, w_dhn, w_part, w_split, w_total;
    size_t split_floats;
    // per-device tiling
    int dev;
    int num_cus;
    bool fwd_ok, bwd_ok;
    RecTiling fwd, bwd;
};

namespace {

thread_local char g_detail[256] = "";

void set_detail(const char *what, hipError_t e)
{
    std::snprintf(g_detail, sizeof(g_detail), "%s: %s", what, hipGetErrorString(e));
}

lstm_status_t hip_status(const char *what, hipError_t e)
{
    if (e == hipSuccess) return LSTM_OK;
    set_detail(what, e);
    if (e == hipErrorCooperativeLaunchTooLarge) return LSTM_ERR_UNSUPPORTED;
    return LSTM_ERR_HIP;
}

lstm_status_t invalid(const char *what)
{
    std::snprintf(g_detail, sizeof(g_detail), "invalid argument: %s", what);
    return LSTM_ERR_INVALID_ARG;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

lstm_status_t short_buffer(const char *what, size_t given, size_t need)
{
    std::snprintf(g_detail, sizeof(g_detail), "%s: %zu bytes given, %zu needed", what, given, need);
    return LSTM_ERR_WORKSPACE;
}
bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

lstm_status_t ensure_plan(lstm_handle *h)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status("hipGetDevice", e);
    if (h->dev == dev) return LSTM_OK;
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_status("hipDeviceGetAttribute", e);
    RecShape sh{h->d.T, h->d.B, h->d.I, h->d.H, h->d.Hp, h->d.reverse, h->ldy};
    h->fwd_ok = plan_forward(h->dt, sh, cus, &h->fwd);
    h->bwd_ok = plan_backward(h->dt, sh, cus, &h->bwd);
    h->num_cus = cus;
    h->dev = dev;
    return LSTM_OK;
}

// Recurrence implementation for this handle: the persistent kernels keep
// the recurrent weights on chip; the stepwise sequence streams them per step
// and is used for LSTMP layers with wide cells (BigLSTM: 8192 cells) and
// whenever no persistent tiling fits.  LSTM355_RECURRENCE=stepwise or
// =persistent overrides the choice (testing and tuning).
bool use_stepwise(const lstm_handle *h, bool persistent_ok)
{
    const char *env = std::getenv("LSTM355_RECURRENCE");
    if (env && std::strcmp(env, "stepwise") == 0) return true;
    if (env && std::strcmp(env, "persistent") == 0 && persistent_ok) return false;
    if (!persistent_ok) return true;
    return h->d.Hp > 0 && h->d.H >= 2048;
}

#define TRY_HIP(what, expr)                                  \
    do {                                                     \
        hipError_t e_ = (expr);                              \
        if (e_ != hipSuccess) return hip_status(what, e_);   \
    } while (0)

}  // namespace

extern "C" const char *lstm_last_error_detail(void) { return g_detail; }

extern "C" const char *lstm_status_string(lstm_status_t s)
{
    switch (s) {
    case LSTM_OK: return "LSTM_OK";
    case LSTM_ERR_INVALID_ARG: return "LSTM_ERR_INVALID_ARG";
    case LSTM_ERR_UNSUPPORTED: return "LSTM_ERR_UNSUPPORTED";
    case LSTM_ERR_WORKSPACE: return "LSTM_ERR_WORKSPACE";
    case LSTM_ERR_HIP: return "LSTM_ERR_HIP";
    case LSTM_ERR_TIMEOUT: return "LSTM_ERR_TIMEOUT";
    }
    return "LSTM_ERR_UNKNOWN";
}

extern "C" lstm_status_t lstm_create(const lstm_desc_t *desc, lstm_handle_t *out)
{
    try {
        if (!desc || !out) return invalid("desc/out is NULL");
        *out = nullptr;
        const lstm_desc_t &d = *desc;
        if (d.T < 1 || d.B < 1 || d.I < 1 || d.H < 1) return invalid("T, B, I, H must be positive");
        if (d.Hp < 0) return invalid("Hp must be >= 0");
        if (d.dtype != LSTM_F32 && d.dtype != LSTM_BF16) return invalid("unknown dtype");
        if (d.reverse != 0 && d.reverse != 1) return invalid("reverse must be 0 or 1");
        if (d.I % 8 || d.H % 8 || d.Hp % 8) return invalid("I, H and Hp must be multiples of 8");
        const int Hr = d.Hp ? d.Hp : d.H;
        const long ldx = d.ldx ? d.ldx : d.I;
        const long ldy = d.ldy ? d.ldy : Hr;
        if (ldx < d.I || ldx % 8) return invalid("ldx must be >= I and a multiple of 8");
        if (ldy < Hr || ldy % 8) return invalid("ldy must be >= the output width and a multiple of 8");
        const long TB = (long)d.T * d.B;
        const long G4 = 4L * d.H;
        if (TB > (1L << 31) / 1 || G4 * (long)(ldx > G4 ? ldx : G4) > (1L << 40) || TB * G4 > (1L << 40))
            return invalid("sizes too large");

        lstm_handle *h = new (std::nothrow) lstm_handle();
        if (!h) return invalid("out of host memory");
        h->d = d;
        h->dt = d.dtype == LSTM_BF16 ? DType::BF16 : DType::F32;
        h->es = dsize(h->dt);
        h->Hr = Hr;
        h->ldx = ldx;
        h->ldy = ldy;
        h->TB = TB;
        h->G4 = G4;
        size_t o = 0;
        h->r_gates = o; o = align256(o + (size_t)TB * G4 * 4);
        h->r_cs = o;    o = align256(o + (size_t)TB * d.H * 4);
        h->r_ms = o;    o = align256(o + (d.Hp ? (size_t)TB * d.H * h->es : 0));
        {   // the fp16 activated gates of the XCD-local kernels, for the layers they keep them in fp16
            const RecShape sh{d.T, d.B, d.I, d.H, d.Hp, d.reverse, ldy};
            const bool act16 = xcd_act16(h->dt, sh);
            h->r_act16 = act16 ? o : 0;
            o = align256(o + (act16 ? (size_t)TB * G4 * 2 : 0));
        }
        h->r_total = o;
        o = 0;
        h->w_sync = o; o = align256(o + SYNC_BYTES);
        h->w_dz = o;   o = align256(o + (size_t)TB * G4 * h->es);
        h->w_rt = o;   o = align256(o + (size_t)Hr * G4 * h->es);
        h->w_pt = o;   o = align256(o + (d.Hp ? (size_t)d.H * d.Hp * h->es : 0));
        h->w_dH = o;   o = align256(o + (d.Hp ? (size_t)TB * d.Hp * h->es : 0));
        h->w_dcn = o;  o = align256(o + (size_t)d.B * d.H * 4);
        h->w_dhn = o;  o = align256(o + (size_t)d.B * d.H * 4);
        {
            size_t pf = colsum_partial_floats((int)TB, (int)G4);
            if (pf < (size_t)8 * G4) pf = (size_t)8 * G4;   // per-XCD bias partials
            h->w_part = o; o = align256(o + pf * 4);
        }
        // split-K partials of the weight- and input-gradient products
        {
            size_t mn = (size_t)G4 * (size_t)(d.I > Hr ? d.I : Hr);
            if (d.Hp && (size_t)d.Hp * d.H > mn) mn = (size_t)d.Hp * d.H;
            h->split_floats = 4 * mn;
        }
        h->w_split = o; o = align256(o + h->split_floats * 4);
        h->w_total = o;
        h->dev = -1;
        h->fwd_ok = h->bwd_ok = false;
        *out = h;
        return LSTM_OK;
    } catch (...) {
        return invalid("exception");
    }
}

extern "C" size_t lstm_reserve_size(lstm_handle_t h) { return h ? h->r_total : 0; }
extern "C" size_t lstm_workspace_size(lstm_handle_t h) { return h ? h->w_total : 0; }

extern "C" lstm_status_t lstm_destroy(lstm_handle_t h)
{
    delete h;
    return LSTM_OK;
}

namespace {
// Validation shared by the forward entry points (everything but the workspace).
lstm_status_t check_forward_args(lstm_handle_t h, const void *x, const void *h0, const float *c0, const void *W,
                                 const void *R, const float *b, const void *P, const void *y, const void *hT,
                                 const float *cT, const void *reserve, size_t reserve_bytes)
{
    if (!h) return invalid("handle is NULL");
    const lstm_desc_t &d = h->d;
    if (!x || !W || !R || !b || !y || !reserve) return invalid("required pointer is NULL");
    if ((P != nullptr) != (d.Hp > 0)) return invalid("P must be given iff Hp > 0");
    for (const void *p : {x, h0, W, R, P, y, hT, reserve})
        if (p && !aligned16(p)) return invalid("device tensors must be 16-byte aligned");
    for (const void *p : {(const void *)c0, (const void *)b, (const void *)cT})
        if (p && !aligned4(p)) return invalid("fp32 tensors must be 4-byte aligned");
    if (reserve_bytes < h->r_total) return short_buffer("reserve", reserve_bytes, h->r_total);
    return LSTM_OK;
}

// One layer's forward pass (arguments validated, plan made): the input
// projection, then the recurrence.  `wv` is the workspace (sync words at
// w_sync; the stepwise recurrence also uses the split-K partials at w_split);
// full_ws: it is the whole workspace, not the allocation-free entry point's
// scratch, so the XCD-local forward may keep an fp16 input projection in it.
lstm_status_t forward_impl(lstm_handle_t h, const void *x, const void *h0, const float *c0, const void *W,
                           const void *R, const float *b, const void *P, void *y, void *hT, float *cT,
                           void *reserve, char *wv, bool full_ws, hipStream_t s)
{
    const lstm_desc_t &d = h->d;
    char *rv = static_cast<char *>(reserve);
    float *gates = reinterpret_cast<float *>(rv + h->r_gates);

    RecShape sh{d.T, d.B, d.I, d.H, d.Hp, d.reverse, h->ldy};
    FwdBufs fb{};
    fb.R = R; fb.P = P; fb.h0 = h0; fb.c0 = c0;
    fb.gates = gates;
    fb.cs = reinterpret_cast<float *>(rv + h->r_cs);
    fb.ms = d.Hp ? rv + h->r_ms : nullptr;
    fb.y = y; fb.hT = hT; fb.cT = cT;
    fb.sync = reinterpret_cast<unsigned *>(wv + h->w_sync);
    const bool xcd = xcd_path_ok(h->dt, sh, h->num_cus);
    if (xcd && h->r_act16) fb.act16 = rv + h->r_act16;

    GemmDesc g{};
    g.in = h->dt; g.out_f32 = true; g.a_kmajor = true; g.b_kmajor = true;
    g.M = (int)h->TB; g.N = (int)h->G4; g.K = d.I;
    g.A = x; g.lda = h->ldx;
    g.B = W; g.ldb = d.I;
    g.C = gates; g.ldc = h->G4;
    g.bias = b; g.beta = 0;
    if (xcd) g.side = xcd_prep_forward(sh, fb);   // the recurrence's exchange rows and flags
    if (xcd && full_ws) {
        // the XCD-local forward takes the input projection in fp16, half the
        // bytes of the product's output and of the recurrence's reads, in the
        // workspace's dz rows (the backward's, unused by the forward)
        GemmDesc g16 = g;
        g16.out_f32 = false; g16.out_f16 = true;
        g16.C = wv + h->w_dz;
        if (gemm_f16_ok(g16)) {
            g = g16;
            fb.gx16 = g16.C;
        }
    }
    TRY_HIP("input projection", gemm(g, s, K_GEMM_GX));

    if (!xcd && use_stepwise(h, h->fwd_ok)) {
        StepwiseArgs sw{R, P, reinterpret_cast<float *>(wv + h->w_split), h->split_floats};
        TRY_HIP("forward recurrence (stepwise)", forward_stepwise(h->dt, sh, fb, sw, s));
    } else if (xcd) {
        TRY_HIP("forward recurrence (XCD-local)", launch_forward_xcd(sh, fb, watchdog_ticks(), s, true));
    } else {
        TRY_HIP("forward recurrence", launch_forward(h->dt, sh, h->fwd, fb, s));
    }
    return LSTM_OK;
}

// Scratch of lstm_forward_noalloc: the sync words (barrier counter, abort
// word, per-XCD claim masks) that the persistent recurrences need, in a
// device array each GPU holds until the process ends.  Host code never uses
// the array's name as an address: its device address is looked up once per
// device with hipGetSymbolAddress and kept in g_scratch_ptr.
constexpr size_t NOALLOC_SCRATCH_BYTES = 64 * 1024;
constexpr int MAX_DEVICES = 64;
}  // namespace

static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device (looked up on first use).
lstm_status_t scratch_address(char **out)
{
    int dev = 0;
    TRY_HIP("hipGetDevice", hipGetDevice(&dev));
    if (dev < 0 || dev >= MAX_DEVICES) return invalid("device ordinal beyond the scratch table");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        TRY_HIP("hipGetSymbolAddress(scratch)", hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
        if (!ptr) return hip_status("hipGetSymbolAddress(scratch)", hipErrorInvalidSymbol);
        g_scratch_ptr[dev] = ptr;
    }
    *out = static_cast<char *>(g_scratch_ptr[dev]);
    return LSTM_OK;
}
}  // namespace

extern "C" lstm_status_t lstm_forward(lstm_handle_t h, const void *x, const void *h0, const float *c0, const void *W,
                                      const void *R, const float *b, const void *P, void *y, void *hT, float *cT,
                                      void *reserve, size_t reserve_bytes, void *workspace, size_t workspace_bytes,
                                      void *stream)
{
    try {
        lstm_status_t st = check_forward_args(h, x, h0, c0, W, R, b, P, y, hT, cT, reserve, reserve_bytes);
        if (st != LSTM_OK) return st;
        if (!workspace) return invalid("required pointer is NULL");
        if (!aligned16(workspace)) return invalid("device tensors must be 16-byte aligned");
        if (workspace_bytes < h->w_total) return short_buffer("workspace", workspace_bytes, h->w_total);
        st = ensure_plan(h);
        if (st != LSTM_OK) return st;
        return forward_impl(h, x, h0, c0, W, R, b, P, y, hT, cT, reserve, static_cast<char *>(workspace), true,
                            static_cast<hipStream_t>(stream));
    } catch (...) {
        return invalid("exception");
    }
}

extern "C" lstm_status_t lstm_forward_noalloc(lstm_handle_t h, const void *x, const void *h0, const float *c0,
                                              const void *W, const void *R, const float *b, const void *P, void *y,
                                              void *hT, float *cT, void *reserve, size_t reserve_bytes, void *stream)
{
    try {
        lstm_status_t st = check_forward_args(h, x, h0, c0, W, R, b, P, y, hT, cT, reserve, reserve_bytes);
        if (st != LSTM_OK) return st;
        st = ensure_plan(h);
        if (st != LSTM_OK) return st;
        // the persistent recurrences need only the sync words; the stepwise
        // sequence (wide LSTMP layers) needs split-K partials as well
        const lstm_desc_t &d = h->d;
        RecShape sh{d.T, d.B, d.I, d.H, d.Hp, d.reverse, h->ldy};
        const bool stepwise = !xcd_path_ok(h->dt, sh, h->num_cus) && use_stepwise(h, h->fwd_ok);
        const size_t need = stepwise ? h->w_split + h->split_floats * 4 : h->w_sync + SYNC_BYTES;
        if (need > NOALLOC_SCRATCH_BYTES) {
            std::snprintf(g_detail, sizeof(g_detail),
                          "lstm_forward_noalloc: this layer needs %zu bytes of scratch, the library holds %zu "
                          "(call lstm_forward with a workspace)", need, NOALLOC_SCRATCH_BYTES);
            return LSTM_ERR_WORKSPACE;
        }
        char *wv = nullptr;
        st = scratch_address(&wv);
        if (st != LSTM_OK) return st;
        return forward_impl(h, x, h0, c0, W, R, b, P, y, hT, cT, reserve, wv, false, static_cast<hipStream_t>(stream));
    } catch (...) {
        return invalid("exception");
    }
}

extern "C" lstm_status_t lstm_forward_stack(int L, const lstm_handle_t *hs, const void *x, const void *const *W,
                                            const void *const *R, const float *const *b, void *const *y,
                                            const int *residual, void *const *ysum, void *const *reserve,
                                            size_t reserve_bytes, void *workspace, size_t workspace_bytes,
                                            void *stream)
{
    try {
        if (L < 1 || !hs || !x || !W || !R || !b || !y || !reserve || !workspace)
            return invalid("required pointer is NULL or L < 1");
        for (int l = 0; l < L; ++l) {
            if (!hs[l] || !W[l] || !R[l] || !b[l] || !y[l] || !reserve[l]) return invalid("required pointer is NULL");
            for (const void *p : {W[l], R[l], (const void *)y[l], (const void *)reserve[l]})
                if (!aligned16(p)) return invalid("device tensors must be 16-byte aligned");
            if (!aligned4(b[l])) return invalid("fp32 tensors must be 4-byte aligned");
        }
        if (!aligned16(x) || !aligned16(workspace)) return invalid("device tensors must be 16-byte aligned");
        if (residual)
            for (int l = 0; l < L; ++l)
                if (residual[l]) {
                    if (!ysum || !ysum[l]) return invalid("a residual layer needs its sum buffer");
                    if (!aligned16(ysum[l])) return invalid("device tensors must be 16-byte aligned");
                    const lstm_desc_t &d = hs[l]->d;
                    if (d.I != d.H || hs[l]->ldx != d.H || hs[l]->ldy != d.H)
                        return invalid("a residual layer needs an input as wide as its output");
                }
        for (int l = 0; l < L; ++l) {
            if (reserve_bytes < hs[l]->r_total) return short_buffer("reserve", reserve_bytes, hs[l]->r_total);
            if (workspace_bytes < hs[l]->w_total) return short_buffer("workspace", workspace_bytes, hs[l]->w_total);
        }
        auto unsupported = [](const char *why) {
            std::snprintf(g_detail, sizeof(g_detail), "layer wavefront not available: %s", why);
            return LSTM_ERR_UNSUPPORTED;
        };
        if (L < 2 || L > 4) return unsupported("needs 2 to 4 layers");
        const lstm_desc_t &d0 = hs[0]->d;
        for (int l = 0; l < L; ++l) {
            const lstm_desc_t &d = hs[l]->d;
            if (hs[l]->dt != DType::BF16 || d.Hp != 0 || d.reverse != 0) return unsupported("bf16 LSTM layers only");
            if (d.T != d0.T || d.B != d0.B || d.H != d0.H) return unsupported("layers differ in T, B or H");
            if (l > 0 && (d.I != d.H || hs[l]->ldx != d.H)) return unsupported("a layer's input is not the layer below");
        }
        for (int l = 0; l < L; ++l) {   // the checks that query the device
            const lstm_desc_t &d = hs[l]->d;
            RecShape sh{d.T, d.B, d.I, d.H, d.Hp, d.reverse, hs[l]->ldy};
            lstm_status_t st = ensure_plan(hs[l]);
            if (st != LSTM_OK) return st;
            if (!wave_path_ok(sh, hs[l]->num_cus)) return unsupported("shape or device");
        }
        hipStream_t s = static_cast<hipStream_t>(stream);
        lstm_handle *h0 = hs[0];
        char *wv = static_cast<char *>(workspace);
        WaveBufs wb[4];
        for (int l = 0; l < L; ++l) {
            char *rv = static_cast<char *>(reserve[l]);
            wb[l].R = R[l];
            wb[l].W = W[l];
            wb[l].bias = b[l];
            wb[l].gates = reinterpret_cast<float *>(rv + hs[l]->r_gates);
            wb[l].cs = reinterpret_cast<float *>(rv + hs[l]->r_cs);
            wb[l].y = y[l];
            wb[l].in_b = nullptr;
            wb[l].sum = nullptr;
            wb[l].poll_b = 0;
        }
        // output of layer l (the input of layer l+1): y_l, or y_l plus the
        // layer's own input for a residual layer
        auto res = [&](int l) { return residual && residual[l]; };
        auto input_of = [&](int l) -> const void * { return l == 0 ? x : (res(l - 1) ? ysum[l - 1] : y[l - 1]); };
        for (int l = 1; l < L; ++l)
            if (res(l - 1)) {   // layer l's projection forms the sum and stores it
                wb[l].in_b = input_of(l - 1);
                wb[l].poll_b = l - 1 > 0;
                wb[l].sum = ysum[l - 1];
            }
        // Layer 0's input projection: inside the wavefront when x has the
        // layers' width (an otherwise idle XCD computes it step by step),
        // else by the GEMM as in lstm_forward.  The other layers' are always
        // computed in the wavefront.
        const bool x_in_wave = d0.I == d0.H && h0->ldx == d0.H;
        if (!x_in_wave) {
            GemmDesc g{};
            g.in = DType::BF16; g.out_f32 = true; g.a_kmajor = true; g.b_kmajor = true;
            g.M = (int)h0->TB; g.N = (int)h0->G4; g.K = d0.I;
            g.A = x; g.lda = h0->ldx;
            g.B = W[0]; g.ldb = d0.I;
            g.C = wb[0].gates; g.ldc = h0->G4;
            g.bias = b[0]; g.beta = 0;
            TRY_HIP("input projection", gemm(g, s, K_GEMM_GX));
        }
        RecShape sh{d0.T, d0.B, d0.I, d0.H, 0, 0, h0->ldy};
        TRY_HIP("layer wavefront", launch_forward_wave(sh, L, x_in_wave ? x : nullptr, wb,
                                                       reinterpret_cast<unsigned *>(wv + h0->w_sync),
                                                       watchdog_ticks(), s));
        if (res(L - 1))   // the top layer's sum: the stack's output
            TRY_HIP("residual sum", add(DType::BF16, (size_t)d0.T * d0.B * d0.H, y[L - 1], input_of(L - 1),
                                        ysum[L - 1], s));
        return LSTM_OK;
    } catch (...) {
        return invalid("exception");
    }
}

namespace {
// Workspace of lstm_backward_stack: flags, then per layer dz and (below the
// top layer) the upstream gradient written inside the launch, then the bias
// gradients.
struct StackBwdLayout {
    size_t sync, dz[4], dy[4], dbp, total;
};

StackBwdLayout stack_bwd_layout(int L, const lstm_desc_t &d)
{
    StackBwdLayout w{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = align256(off + bytes);
        return o;
    };
    const size_t H = (size_t)d.H, TB = (size_t)d.T * d.B;
    w.sync = take((size_t)(XCD_FLAGS + XCD_WORDS) * 4);
    for (int l = 0; l < L; ++l) {
        w.dz[l] = take(TB * 4 * H * 2);
        w.dy[l] = l < L - 1 ? take(TB * H * 2) : 0;
    }
    w.dbp = take((size_t)L * 4 * H * 4);
    w.total = off;
    return w;
}

// Descriptor-level conditions of the backward layer wavefront (no device query).
const char *stack_bwd_unfit(int L, const lstm_handle_t *hs)
{
    if (L < 2 || L > 4) return "needs 2 to 4 layers";
    const lstm_desc_t &d0 = hs[0]->d;
    if (d0.T < 2) return "needs T >= 2";
    for (int l = 0; l < L; ++l) {
        const lstm_desc_t &d = hs[l]->d;
        if (hs[l]->dt != DType::BF16 || d.Hp != 0 || d.reverse != 0) return "bf16 LSTM layers only";
        if (d.T != d0.T || d.B != d0.B || d.H != d0.H) return "layers differ in T, B or H";
        if (d.I != d.H || hs[l]->ldx != d.H || hs[l]->ldy != d.H) return "every layer needs I = H and dense x, y";
    }
    return nullptr;
}
}  // namespace

extern "C" size_t lstm_backward_stack_workspace_size(int L, const lstm_handle_t *hs)
{
    if (!hs || L < 1) return 0;
    for (int l = 0; l < L; ++l)
        if (!hs[l]) return 0;
    if (stack_bwd_unfit(L, hs)) return 0;
    return stack_bwd_layout(L, hs[0]->d).total;
}

extern "C" lstm_status_t lstm_backward_stack(int L, const lstm_handle_t *hs, const void *dy, const void *x,
                                             const void *const *W, const void *const *R, const void *const *y,
                                             const int *residual, const void *const *ysum,
                                             const void *const *reserve, size_t reserve_bytes, void *dx,
                                             float *const *dW, float *const *dR, float *const *db, int accumulate,
                                             void *workspace, size_t workspace_bytes, void *stream)
{
    try {
        if (L < 1 || !hs || !dy || !x || !W || !R || !y || !reserve || !dW || !dR || !db || !workspace)
            return invalid("required pointer is NULL or L < 1");
        if (accumulate != 0 && accumulate != 1) return invalid("accumulate must be 0 or 1");
        for (int l = 0; l < L; ++l) {
            if (!hs[l] || !W[l] || !R[l] || !y[l] || !reserve[l] || !dW[l] || !dR[l] || !db[l])
                return invalid("required pointer is NULL");
            for (const void *p : {W[l], R[l], y[l], reserve[l]})
                if (!aligned16(p)) return invalid("device tensors must be 16-byte aligned");
            for (const void *p : {(const void *)dW[l], (const void *)dR[l], (const void *)db[l]})
                if (!aligned4(p)) return invalid("fp32 tensors must be 4-byte aligned");
        }
        for (const void *p : {dy, x, (const void *)dx, (const void *)workspace})
            if (p && !aligned16(p)) return invalid("device tensors must be 16-byte aligned");
        auto res = [&](int l) { return residual && residual[l]; };
        for (int l = 0; l < L - 1; ++l)   // the sums that feed the layers above (the weight gradients' inputs)
            if (res(l) && (!ysum || !ysum[l] || !aligned16(ysum[l])))
                return invalid("a residual layer needs its 16-byte aligned sum buffer");
        if (const char *why = stack_bwd_unfit(L, hs)) {
            std::snprintf(g_detail, sizeof(g_detail), "layer wavefront not available: %s", why);
            return LSTM_ERR_UNSUPPORTED;
        }
        for (int l = 0; l < L; ++l)
            if (reserve_bytes < hs[l]->r_total) return short_buffer("reserve", reserve_bytes, hs[l]->r_total);
        {
            const size_t need = stack_bwd_layout(L, hs[0]->d).total;
            if (workspace_bytes < need) return short_buffer("workspace", workspace_bytes, need);
        }
        const lstm_desc_t &d0 = hs[0]->d;
        const int T = d0.T, B = d0.B, H = d0.H;
        const long G4 = 4L * H, TB = (long)T * B;
        for (int l = 0; l < L; ++l) {   // the checks that query the device
            lstm_status_t st = ensure_plan(hs[l]);
            if (st != LSTM_OK) return st;
            RecShape sh{T, B, H, H, 0, 0, hs[l]->ldy};
            if (!wave_path_ok(sh, hs[l]->num_cus)) {
                std::snprintf(g_detail, sizeof(g_detail), "layer wavefront not available: shape or device");
                return LSTM_ERR_UNSUPPORTED;
            }
        }
        const StackBwdLayout lay = stack_bwd_layout(L, d0);
        char *wv = static_cast<char *>(workspace);
        // [dW | dR] of every layer as one product each (checked before anything runs)
        GemmDesc gw[4];
        for (int l = 0; l < L; ++l) {
            GemmDesc &g = gw[l];
            g = GemmDesc{};
            g.in = DType::BF16; g.out_f32 = true; g.a_kmajor = false; g.b_kmajor = false;
            g.M = (int)G4; g.N = 2 * H; g.K = (int)TB;
            g.A = wv + lay.dz[l]; g.lda = G4;
            g.B = l == 0 ? x : (res(l - 1) ? ysum[l - 1] : y[l - 1]); g.ldb = H;
            g.C = dW[l]; g.ldc = H; g.beta = accumulate;
            g.N1 = H;
            g.B2 = y[l]; g.ldb2 = H; g.b2_bytes = TB * H * 2;   // dz_t pairs with y_{t-1}; h0 is zero
            g.ylo = B; g.yhi = (int)TB; g.yoff = -B; g.hlo = 0; g.hlen = B;
            g.C2 = dR[l]; g.ldc2 = H;
            g.side.sum_src = reinterpret_cast<const float *>(wv + lay.dbp) + (size_t)l * G4;
            g.side.sum_rows = 1;
            g.side.sum_cols = (int)G4;
            g.side.sum_dst = db[l];
            g.side.sum_acc = accumulate;
            if (!gemm_dual_ok(g)) {
                std::snprintf(g_detail, sizeof(g_detail), "layer wavefront not available: weight-gradient shape");
                return LSTM_ERR_UNSUPPORTED;
            }
        }
        hipStream_t s = static_cast<hipStream_t>(stream);
        WaveBwdBufs wb[4];
        for (int l = 0; l < L; ++l) {
            const char *rv = static_cast<const char *>(reserve[l]);
            const bool want_dx = l > 0 || dx;
            wb[l].R = R[l];
            wb[l].W = want_dx ? W[l] : nullptr;
            wb[l].gates = reinterpret_cast<const float *>(rv + hs[l]->r_gates);
            wb[l].cs = reinterpret_cast<const float *>(rv + hs[l]->r_cs);
            wb[l].dz = wv + lay.dz[l];
            wb[l].dy = l == L - 1 ? dy : wv + lay.dy[l];
            wb[l].dy_fill = l == L - 1 ? nullptr : wv + lay.dy[l];
            wb[l].dx = l == 0 ? dx : wv + lay.dy[l - 1];
            wb[l].dbp = reinterpret_cast<float *>(wv + lay.dbp) + (size_t)l * G4;
            wb[l].residual = res(l) ? 1 : 0;
        }
        // one launch arms the rows the wavefront exchanges, then the wavefront
        // itself (its workgroups read the columns of R and W they keep)
        RecShape sh{T, B, H, H, 0, 0, hs[0]->ldy};
        unsigned *sync = reinterpret_cast<unsigned *>(wv + lay.sync);
        TRY_HIP("layer wavefront (backward)", launch_backward_wave(sh, L, wb, sync, watchdog_ticks(), s, false));
        // the layers' weight-gradient products as one batched launch
        GemmDesc gb = gw[0];
        gb.nbatch = L;
        gb.batch = gw;
        TRY_HIP("dW|dR", gemm(gb, s, K_GEMM_DWR));
        return LSTM_OK;
    } catch (...) {
        return invalid("exception");
    }
}

extern "C" lstm_status_t lstm_backward(lstm_handle_t h, const void *dy, const void *dhT, const float *dcT,
                                       const void *x, const void *h0, const float *c0, const void *W, const void *R,
                                       const void *P, const void *y, const void *reserve, size_t reserve_bytes,
                                       void *dx, void *dh0, float *dc0, float *dW, float *dR, float *db, float *dP,
                                       int accumulate, void *workspace, size_t workspace_bytes, void *stream)
{
    try {
        if (!h) return invalid("handle is NULL");
        const lstm_desc_t &d = h->d;
        if (!dy || !x || !W || !R || !y || !reserve || !workspace || !dW || !dR || !db)
            return invalid("required pointer is NULL");
        if ((P != nullptr) != (d.Hp > 0)) return invalid("P must be given iff Hp > 0");
        if (d.Hp > 0 && !dP) return invalid("dP is required for LSTMP");
        if (accumulate != 0 && accumulate != 1) return invalid("accumulate must be 0 or 1");
        for (const void *p : {dy, dhT, x, h0, W, R, P, y, reserve, (const void *)dx, (const void *)dh0, (const void *)workspace})
            if (p && !aligned16(p)) return invalid("device tensors must be 16-byte aligned");
        for (const void *p : {(const void *)dcT, (const void *)c0, (const void *)dc0, (const void *)dW,
                              (const void *)dR, (const void *)db, (const void *)dP})
            if (p && !aligned4(p)) return invalid("fp32 tensors must be 4-byte aligned");
        if (reserve_bytes < h->r_total) return short_buffer("reserve", reserve_bytes, h->r_total);
        if (workspace_bytes < h->w_total) return short_buffer("workspace", workspace_bytes, h->w_total);
        lstm_status_t st = ensure_plan(h);
        if (st != LSTM_OK) return st;
        hipStream_t s = static_cast<hipStream_t>(stream);
        const char *rv = static_cast<const char *>(reserve);
        char *wv = static_cast<char *>(workspace);
        const int T = d.T, B = d.B, I = d.I, H = d.H, Hp = d.Hp, Hr = h->Hr;
        const long G4 = h->G4, TB = h->TB;
        const size_t es = h->es;
        void *dz = wv + h->w_dz;
        void *Rt = wv + h->w_rt;
        void *Pt = Hp ? wv + h->w_pt : nullptr;
        void *dH = Hp ? wv + h->w_dH : nullptr;
        float *split_ws = reinterpret_cast<float *>(wv + h->w_split);

        RecShape sh{T, B, I, H, Hp, d.reverse, h->ldy};
        const bool xcd = xcd_path_ok(h->dt, sh, h->num_cus);
        const bool stepwise = !xcd && use_stepwise(h, h->bwd_ok);

        BwdBufs bb{};
        bb.Rt = Rt; bb.Pt = Pt; bb.dy = dy; bb.dhT = dhT; bb.dcT = dcT; bb.h0 = h0; bb.c0 = c0;
        bb.gates = reinterpret_cast<const float *>(rv + h->r_gates);
        bb.act16 = (xcd && h->r_act16) ? rv + h->r_act16 : nullptr;
        bb.cs = reinterpret_cast<const float *>(rv + h->r_cs);
        bb.dz = dz; bb.dH = dH;
        bb.dcn = reinterpret_cast<float *>(wv + h->w_dcn);
        bb.dhn = reinterpret_cast<float *>(wv + h->w_dhn);
        bb.dh0 = dh0; bb.dc0 = dc0;
        bb.dbpart = reinterpret_cast<float *>(wv + h->w_part);
        bb.sync = reinterpret_cast<unsigned *>(wv + h->w_sync);
        if (!stepwise) {   // the persistent kernels keep rows of R^T (and P^T)
            // (reading R's columns in the kernel instead measured slower here:
            // the transpose hides behind the exchange fill it carries)
            const SideJob prep = xcd ? xcd_prep_backward(sh, bb) : SideJob{};
            TRY_HIP("transpose R", transpose(h->dt, R, (int)G4, Hr, Rt, s, xcd ? &prep : nullptr));
            if (Hp) TRY_HIP("transpose P", transpose(h->dt, P, Hp, H, Pt, s));
        }
        if (stepwise) {
            StepwiseArgs sw{R, P, split_ws, h->split_floats};
            TRY_HIP("backward recurrence (stepwise)", backward_stepwise(h->dt, sh, bb, sw, s));
        } else if (xcd) {
            TRY_HIP("backward recurrence (XCD-local)", launch_backward_xcd(sh, bb, watchdog_ticks(), s, true));
        } else {
            TRY_HIP("backward recurrence", launch_backward(h->dt, sh, h->bwd, bb, s));
        }

        if (dx) {  // dX = dZ W
            GemmDesc g{};
            g.in = h->dt; g.out_f32 = h->dt == DType::F32; g.a_kmajor = true; g.b_kmajor = false;
            g.M = (int)TB; g.N = I; g.K = (int)G4;
            g.A = dz; g.lda = G4; g.B = W; g.ldb = I; g.C = dx; g.ldc = h->ldx;
            // few output tiles over a long K (small batches, wide layers): split K
            g.splitk_ws = split_ws; g.splitk_ws_floats = h->split_floats;
            TRY_HIP("dx", gemm(g, s, K_GEMM_DX));
        }
        // [dW | dR] = dZ^T [X | H_prev] as one product when the shapes allow
        // (H_prev: y of the previous visited step, h0 for the first one)
        bool fused = false;
        if (h->dt == DType::BF16 && (B % 32 == 0 || !h0) && T > 1) {
            GemmDesc g{};
            g.in = h->dt; g.out_f32 = true; g.a_kmajor = false; g.b_kmajor = false;
            g.M = (int)G4; g.N = I + Hr; g.K = (int)TB;
            g.A = dz; g.lda = G4; g.B = x; g.ldb = h->ldx; g.C = dW; g.ldc = I; g.beta = accumulate;
            g.N1 = I;
            g.B2 = y; g.ldb2 = h->ldy; g.b2_bytes = (long)TB * h->ldy * (long)es;
            g.B3 = h0; g.ldb3 = Hr; g.b3_bytes = (long)B * Hr * (long)es;
            if (!d.reverse) {   // k = t*B + b pairs dz_t with y_{t-1} (t >= 1), h0 (t = 0)
                g.ylo = B; g.yhi = (int)TB; g.yoff = -B; g.hlo = 0;
            } else {            // dz_t with y_{t+1} (t <= T-2), h0 (t = T-1)
                g.ylo = 0; g.yhi = (int)TB - B; g.yoff = B; g.hlo = (int)TB - B;
            }
            g.hlen = B;
            g.C2 = dR; g.ldc2 = Hr;
            if (xcd) {   // db = sum of the recurrence's per-XCD partials, done by the same launch
                g.side.sum_src = reinterpret_cast<const float *>(wv + h->w_part);
                g.side.sum_rows = 8;
                g.side.sum_cols = (int)G4;
                g.side.sum_dst = db;
                g.side.sum_acc = accumulate;
            }
            if (gemm_dual_ok(g)) {
                TRY_HIP("dW|dR", gemm(g, s, K_GEMM_DWR));
                fused = true;
            }
        }
        if (!fused) {  // dW = dZ^T X
            GemmDesc g{};
            g.in = h->dt; g.out_f32 = true; g.a_kmajor = false; g.b_kmajor = false;
            g.M = (int)G4; g.N = I; g.K = (int)TB;
            g.A = dz; g.lda = G4; g.B = x; g.ldb = h->ldx; g.C = dW; g.ldc = I; g.beta = accumulate;
            g.splitk_ws = split_ws; g.splitk_ws_floats = h->split_floats;
            TRY_HIP("dW", gemm(g, s, K_GEMM_DW));
        }
        if (!fused) {  // dR = sum_t dz_t^T h_{t-1}: steps after the first see y of the previous step, the first sees h0
            int beta = accumulate;
            const char *dzc = static_cast<const char *>(dz);
            const char *yc = static_cast<const char *>(y);
            if (T > 1) {
                GemmDesc g{};
                g.in = h->dt; g.out_f32 = true; g.a_kmajor = false; g.b_kmajor = false;
                g.M = (int)G4; g.N = Hr; g.K = (T - 1) * B;
                if (!d.reverse) {
                    g.A = dzc + (size_t)B * G4 * es;   // dz at t = 1 .. T-1
                    g.B = yc;                          // y  at t = 0 .. T-2
                } else {
                    g.A = dzc;                                  // dz at t = 0 .. T-2
                    g.B = yc + (size_t)B * h->ldy * es;         // y  at t = 1 .. T-1
                }
                g.lda = G4; g.ldb = h->ldy; g.C = dR; g.ldc = Hr; g.beta = beta;
                g.splitk_ws = split_ws; g.splitk_ws_floats = h->split_floats;
                TRY_HIP("dR", gemm(g, s, K_GEMM_DR));
                beta = 1;
            }
            if (h0) {
                const int tf = d.reverse ? T - 1 : 0;
                GemmDesc g{};
                g.in = h->dt; g.out_f32 = true; g.a_kmajor = false; g.b_kmajor = false;
                g.M = (int)G4; g.N = Hr; g.K = B;
                g.A = dzc + (size_t)tf * B * G4 * es; g.lda = G4;
                g.B = h0; g.ldb = Hr; g.C = dR; g.ldc = Hr; g.beta = beta;
                TRY_HIP("dR(h0)", gemm(g, s, K_GEMM_DR));
                beta = 1;
            }
            if (!beta) TRY_HIP("dR zero", fill_u32(dR, (size_t)G4 * Hr, 0u, s));
        }
        if (xcd) {   // the recurrence left one fp32 partial per XCD (the fused product sums them itself)
            if (!fused)
                TRY_HIP("db", sum_rows(reinterpret_cast<const float *>(wv + h->w_part), 8, (int)G4, db, accumulate, s));
        } else
            TRY_HIP("db", colsum(h->dt, dz, (int)TB, (int)G4, reinterpret_cast<float *>(wv + h->w_part), db, accumulate, s));
        if (Hp) {  // dP = sum_t dh_t^T m_t
            GemmDesc g{};
            g.in = h->dt; g.out_f32 = true; g.a_kmajor = false; g.b_kmajor = false;
            g.M = Hp; g.N = H; g.K = (int)TB;
            g.A = dH; g.lda = Hp; g.B = rv + h->r_ms; g.ldb = H; g.C = dP; g.ldc = H; g.beta = accumulate;
            g.splitk_ws = split_ws; g.splitk_ws_floats = h->split_floats;
            TRY_HIP("dP", gemm(g, s, K_GEMM_DP));
        }
        return LSTM_OK;
    } catch (...) {
        return invalid("exception");
    }
}

extern "C" lstm_status_t lstm_check(lstm_handle_t h, void *workspace, void *stream)
{
    (void)workspace;   // the trip flags are per device, not per workspace
    if (!h) return invalid("handle is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    TRY_HIP("stream sync", hipStreamSynchronize(s));
    unsigned tripped = 0;
    unsigned tripped_xcd = 0;
    TRY_HIP("read watchdog flag", watchdog_read_and_clear(&tripped));
    TRY_HIP("read watchdog flag", xcd_tripped_read_and_clear(&tripped_xcd));
    tripped |= tripped_xcd;
    if (tripped & TRIP_PLACEMENT) {
        // workgroups were not spread over the XCDs as the XCD-local kernels
        // require: stop using them in this process
        xcd_path_disable();
        std::snprintf(g_detail, sizeof(g_detail), "XCD-local kernel did not get one workgroup per (XCD, slot); "
                                                  "falling back to the generic kernels from now on");
        return LSTM_ERR_UNSUPPORTED;
    }
    if (tripped) {
        std::snprintf(g_detail, sizeof(g_detail), "a grid barrier's watchdog expired");
        return LSTM_ERR_TIMEOUT;
    }
    return LSTM_OK;
}

extern "C" lstm_status_t lstm_add(lstm_dtype_t dtype, size_t n, const void *a, const void *b, void *out, void *stream)
{
    if (dtype != LSTM_F32 && dtype != LSTM_BF16) return invalid("unknown dtype");
    if (n == 0) return LSTM_OK;
    if (!a || !b || !out) return invalid("NULL pointer");
    TRY_HIP("add", add(dtype == LSTM_BF16 ? DType::BF16 : DType::F32, n, a, b, out, static_cast<hipStream_t>(stream)));
    return LSTM_OK;
}

/* Tiling chosen for this handle on the current device (diagnostics). */
extern "C" lstm_status_t lstm_describe_tiling(lstm_handle_t h, int *out8)
{
    if (!h || !out8) return invalid("NULL pointer");
    lstm_status_t st = ensure_plan(h);
    if (st != LSTM_OK) return st;
    RecShape sh{h->d.T, h->d.B, h->d.I, h->d.H, h->d.Hp, h->d.reverse, h->ldy};
    const bool xcd = xcd_path_ok(h->dt, sh, h->num_cus);
    if (!xcd && use_stepwise(h, h->fwd_ok && h->bwd_ok)) {
        // stepwise sequence: GEMM launches per step, no persistent grid
        const int v[8] = {0, 0, h->d.B, STEPWISE_VARIANT, 0, 0, h->d.B, STEPWISE_VARIANT};
        for (int i = 0; i < 8; ++i) out8[i] = v[i];
        return LSTM_OK;
    }
    if (xcd) {
        // XCD-local kernels: 256 workgroups, H/32 cells each, ceil(B/8) rows per XCD
        const int rx = (h->d.B + 7) / 8;
        const int v[8] = {256, h->d.H / 32, rx, XCD_VARIANT, 256, h->d.H / 32, rx, XCD_VARIANT};
        for (int i = 0; i < 8; ++i) out8[i] = v[i];
        return LSTM_OK;
    }
    out8[0] = h->fwd_ok ? h->fwd.G : 0;
    out8[1] = h->fwd.HN;
    out8[2] = h->fwd.BM;
    out8[3] = h->fwd.variant;
    out8[4] = h->bwd_ok ? h->bwd.G : 0;
    out8[5] = h->bwd.HN;
    out8[6] = h->bwd.BM;
    out8[7] = h->bwd.variant;
    return LSTM_OK;
}
