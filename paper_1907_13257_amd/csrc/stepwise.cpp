// stepwise.cpp -- the recurrences as a sequence of launches per step, for
// layers whose recurrent weights cannot stay resident on the chip across a
// persistent kernel (BigLSTM's LSTMP layer: R is 32768 x 1024 and P is
// 1024 x 8192, 80 MiB in bf16).
//
// Forward, per visited step t (previous visited step t'):
//   gates_t += h_{t'} R^T        matrix-core GEMM, accumulated onto the input
//                                projection already stored in gates_t
//   cell update                  pointwise: activations in place, c_t, m_t
//                                (LSTMP in bf16: in the GEMM's epilogue)
//   h_t = P m_t (LSTMP)          GEMM (split over k), written into y_t
// Backward, steps in reverse visiting order:
//   dm = P^T dh_t (LSTMP)        GEMM; dh_t = dy_t + P-side carry, kept in dH
//   gate gradients               pointwise: dz_t, the dc carry
//   carry to t' = R^T dz_t       GEMM: into dH_{t'} (LSTMP, on top of dy_{t'})
//                                or into the fp32 dh carry (LSTM)
// The products are the library's GEMM kernels; each launch reads its weights
// from HBM (or the memory-side cache), so a step costs roughly one pass over
// R and P.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace lstm355 {

namespace {

#define RET_IF(expr)                           \
    do {                                       \
        hipError_t e_ = (expr);                \
        if (e_ != hipSuccess) return e_;       \
    } while (0)

GemmDesc base_desc(DType t, const StepwiseArgs &w)
{
    GemmDesc g{};
    g.in = t;
    g.splitk_ws = w.splitk_ws;
    g.splitk_ws_floats = w.splitk_ws_floats;
    return g;
}

}  // namespace

hipError_t forward_stepwise(DType t, const RecShape &sh, const FwdBufs &b, const StepwiseArgs &w, hipStream_t s)
{
    const int T = sh.T, B = sh.B, H = sh.H, Hp = sh.Hp, Hr = Hp ? Hp : H;
    const long G4 = 4L * H;
    const size_t es = dsize(t);
    char *y = static_cast<char *>(b.y);
    int tprev = -1;
    for (int st = 0; st < T; ++st) {
        const int tt = sh.reverse ? T - 1 - st : st;
        const bool last = st == T - 1;
        float *gates_t = b.gates + (long)tt * B * G4;
        const void *hprev = st > 0 ? static_cast<const void *>(y + (long)tprev * B * sh.ldy * es) : b.h0;
        const float *cprev = st > 0 ? b.cs + (long)tprev * B * H : b.c0;
        float *c_t = b.cs + (long)tt * B * H;
        char *y_t = y + (long)tt * B * sh.ldy * es;
        char *m_t = Hp ? static_cast<char *>(b.ms) + (long)tt * B * H * es : nullptr;
        bool cell_done = false;
        if (hprev) {   // z_t = Gx_t + h_{t'} R^T
            GemmDesc g = base_desc(t, w);
            g.out_f32 = true; g.a_kmajor = true; g.b_kmajor = true;
            g.M = B; g.N = (int)G4; g.K = Hr;
            g.A = hprev; g.lda = st > 0 ? sh.ldy : Hr;
            g.B = w.R; g.ldb = Hr;
            g.C = gates_t; g.ldc = G4; g.beta = 1;
            if (Hp) {   // the cell update in the product's epilogue when it fits
                GemmDesc f = g;
                f.cell_h = H; f.cell_prev = cprev; f.cell_c = c_t; f.cell_m = m_t; f.cell_ldm = H;
                f.cell_cT = last ? b.cT : nullptr;
                if (gemm_cell_ok(f)) {
                    RET_IF(gemm(f, s, K_REC_FWD));
                    cell_done = true;
                }
            }
            if (!cell_done) RET_IF(gemm(g, s, K_REC_FWD));
        }
        if (Hp) {
            if (!cell_done)
                RET_IF(gates_forward(t, B, H, gates_t, cprev, c_t, m_t, H, nullptr, 0, last ? b.cT : nullptr, K_REC_FWD,
                                     s));
            GemmDesc g = base_desc(t, w);   // h_t = P m_t
            g.out_f32 = t == DType::F32; g.a_kmajor = true; g.b_kmajor = true;
            g.M = B; g.N = Hp; g.K = H;
            g.A = m_t; g.lda = H;
            g.B = w.P; g.ldb = H;
            g.C = y_t; g.ldc = sh.ldy;
            RET_IF(gemm(g, s, K_REC_FWD));
            if (last && b.hT) RET_IF(copy_rows(t, B, Hp, y_t, sh.ldy, b.hT, Hp, s));
        } else {
            RET_IF(gates_forward(t, B, H, gates_t, cprev, c_t, y_t, sh.ldy, last ? b.hT : nullptr, H,
                                 last ? b.cT : nullptr, K_REC_FWD, s));
        }
        tprev = tt;
    }
    return hipSuccess;
}

hipError_t backward_stepwise(DType t, const RecShape &sh, const BwdBufs &b, const StepwiseArgs &w, hipStream_t s)
{
    const int T = sh.T, B = sh.B, H = sh.H, Hp = sh.Hp, Hr = Hp ? Hp : H;
    const long G4 = 4L * H;
    const size_t es = dsize(t);
    // cell-gradient carry into the last visited step
    if (b.dcT)
        RET_IF(hipMemcpyAsync(b.dcn, b.dcT, (size_t)B * H * 4, hipMemcpyDeviceToDevice, s));
    else
        RET_IF(fill_u32(b.dcn, (size_t)B * H, 0u, s));
    char *dH = static_cast<char *>(b.dH);
    if (Hp) {   // dH_t = dy_t for every step; the carries are added on top
        RET_IF(copy_rows(t, (long)T * B, Hp, b.dy, sh.ldy, dH, Hp, s));
        if (b.dhT) {
            char *dH_last = dH + (long)(sh.reverse ? 0 : T - 1) * B * Hp * es;
            RET_IF(add(t, (size_t)B * Hp, dH_last, b.dhT, dH_last, s));
        }
    }
    for (int st = T - 1; st >= 0; --st) {
        const int tt = sh.reverse ? T - 1 - st : st;
        const int tp = sh.reverse ? tt + 1 : tt - 1;   // previous visited step (st > 0)
        const float *gates_t = b.gates + (long)tt * B * G4;
        const float *c_t = b.cs + (long)tt * B * H;
        const float *cprev = st > 0 ? b.cs + (long)tp * B * H : b.c0;
        char *dz_t = static_cast<char *>(b.dz) + (long)tt * B * G4 * es;
        float *dc0 = st == 0 ? b.dc0 : nullptr;
        if (Hp) {
            GemmDesc g = base_desc(t, w);   // dm = P^T dh_t, rows of dH times P
            g.out_f32 = true; g.a_kmajor = true; g.b_kmajor = false;
            g.M = B; g.N = H; g.K = Hp;
            g.A = dH + (long)tt * B * Hp * es; g.lda = Hp;
            g.B = w.P; g.ldb = H;
            g.C = b.dhn; g.ldc = H;
            // bf16: two halves of k on twice the workgroups (a few batch rows
            // and no split give one workgroup per two CUs), their fp32 sums
            // added by the gate gradients
            const bool halves = t == DType::BF16 && Hp % 128 == 0 && w.splitk_ws &&
                                w.splitk_ws_floats >= 2 * (size_t)B * H;
            if (halves) g.partials = 2;
            RET_IF(gemm(g, s, K_REC_BWD));
            const float *dm0 = halves ? w.splitk_ws : b.dhn;
            const float *dm1 = halves ? w.splitk_ws + (size_t)B * H : nullptr;
            RET_IF(gates_backward(t, B, H, dm0, nullptr, 0, dm1, nullptr, gates_t, c_t, cprev, b.dcn, dz_t, dc0,
                                  K_REC_BWD, s));
        } else {
            const bool first = st == T - 1;
            const char *dy_t = static_cast<const char *>(b.dy) + (long)tt * B * sh.ldy * es;
            RET_IF(gates_backward(t, B, H, nullptr, dy_t, sh.ldy, first ? nullptr : b.dhn, first ? b.dhT : nullptr,
                                  gates_t, c_t, cprev, b.dcn, dz_t, dc0, K_REC_BWD, s));
        }
        if (st > 0 || b.dh0) {   // R^T dz_t: the recurrent gradient of the previous visited step
            GemmDesc g = base_desc(t, w);
            g.a_kmajor = true; g.b_kmajor = false;
            g.M = B; g.N = Hr; g.K = (int)G4;
            g.A = dz_t; g.lda = G4;
            g.B = w.R; g.ldb = Hr;
            if (st == 0) {
                g.out_f32 = t == DType::F32; g.C = b.dh0; g.ldc = Hr;
            } else if (Hp) {
                g.out_f32 = t == DType::F32; g.C = dH + (long)tp * B * Hp * es; g.ldc = Hp; g.beta = 1;
            } else {
                g.out_f32 = true; g.C = b.dhn; g.ldc = H;
            }
            RET_IF(gemm(g, s, K_REC_BWD));
        }
    }
    return hipSuccess;
}

}  // namespace lstm355
