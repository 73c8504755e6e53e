/*
 * lstm_oracle.c -- plain fp64 reference for one LSTM / LSTMP layer:
 * forward pass and back-propagation through time.
 *
 * TEST INFRASTRUCTURE.  Only the tests, the smoke check and the CPU-baseline
 * leg of the benchmark load this file's library.  It shares no code with the
 * GPU path.  Slow on purpose: plain loops, double precision, no blocking.
 * OpenMP only distributes independent output elements over threads; every sum
 * runs in the same order whatever the thread count.
 *
 * What it computes.  The paper (Section 2, "Background") frames a training
 * step as a forward pass over one worker's mini-batch followed by a backward
 * pass that yields the gradients the workers then all-reduce.  For the two
 * recurrent networks of Section 4 (GNMT: LSTM layers of 1024; BigLSTM: LSTM
 * layers of 8192 cells with a 1024-wide projection) the paper names the
 * networks and widths but prints no cell equations, so the cell is the
 * textbook LSTM without peepholes, gate blocks ordered (i, f, g, o):
 *
 *   z_t = W x_t + R h_{t-1} + b                      z = [z_i z_f z_g z_o]
 *   i = sig(z_i)  f = sig(z_f)  g = tanh(z_g)  o = sig(z_o)
 *   c_t = f * c_{t-1} + i * g
 *   m_t = o * tanh(c_t)
 *   h_t = m_t            (LSTM)     or     h_t = P m_t      (LSTMP)
 *   y_t = h_t
 *
 * With `reverse` the layer visits t = T-1 .. 0 (the backward direction of a
 * bidirectional layer); the final state is the one after the last visited t.
 *
 * Backward: the gradient of L = sum_t <dy_t, y_t> + <dhT, h_final>
 * + <dcT, c_final>, summed over the batch, by the chain rule run backwards
 * over the visited steps.
 *
 * Layouts (row-major, dense): x[T][B][I], y[T][B][Hr], h0[B][Hr], c0[B][H],
 * W[4H][I], R[4H][Hr], b[4H], P[Hp][H]; Hr = Hp if Hp > 0 else H.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double sigm(double u)
{
    /* logistic function, evaluated without overflow for either sign */
    if (u >= 0.0)
        return 1.0 / (1.0 + exp(-u));
    double e = exp(u);
    return e / (1.0 + e);
}

int lstm_oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count of the loops below (timing only; the results do not depend
 * on it: every output element is summed by one thread in a fixed order). */
void lstm_oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Time index of the s-th visited step. */
static long step_time(int s, int T, int reverse) { return reverse ? (long)(T - 1 - s) : (long)s; }

/*
 * Forward pass.  Optional outputs (NULL = not wanted): hT[B][Hr], cT[B][H],
 * gates[T][B][4H] (activated i, f, g, o), cs[T][B][H] (c_t), ms[T][B][H] (m_t).
 * h0 / c0 NULL mean zeros.  Returns 0, or -1 on bad sizes / allocation failure.
 */
int lstm_oracle_forward(int T, int B, int I, int H, int Hp, int reverse,
                        const double *x, const double *h0, const double *c0,
                        const double *W, const double *R, const double *b, const double *P,
                        double *y, double *hT, double *cT,
                        double *gates, double *cs, double *ms)
{
    if (T < 1 || B < 1 || I < 1 || H < 1 || Hp < 0 || (Hp > 0 && !P))
        return -1;
    const long Hr = Hp ? Hp : H;
    const long G = 4L * H;
    double *z = malloc(sizeof(double) * (size_t)B * G);      /* pre-activations of this step */
    double *m = malloc(sizeof(double) * (size_t)B * H);      /* o * tanh(c) of this step */
    double *c = malloc(sizeof(double) * (size_t)B * H);      /* running cell state */
    double *hp = malloc(sizeof(double) * (size_t)B * Hr);    /* h_{t-1} */
    if (!z || !m || !c || !hp) {
        free(z); free(m); free(c); free(hp);
        return -1;
    }
    for (long i = 0; i < (long)B * H; ++i) c[i] = c0 ? c0[i] : 0.0;
    for (long i = 0; i < (long)B * Hr; ++i) hp[i] = h0 ? h0[i] : 0.0;

    for (int s = 0; s < T; ++s) {
        const long t = step_time(s, T, reverse);
        const double *xt = x + t * B * I;
        double *yt = y + t * B * Hr;

        /* z = W x_t + R h_{t-1} + b */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long r = 0; r < G; ++r) {
                double acc = b[r];
                for (long k = 0; k < I; ++k) acc += W[r * I + k] * xt[bb * I + k];
                for (long k = 0; k < Hr; ++k) acc += R[r * Hr + k] * hp[bb * Hr + k];
                z[bb * G + r] = acc;
            }

        /* gates, cell update, cell output */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long j = 0; j < H; ++j) {
                const double *zb = z + bb * G;
                double ig = sigm(zb[j]);
                double fg = sigm(zb[H + j]);
                double gg = tanh(zb[2 * H + j]);
                double og = sigm(zb[3 * H + j]);
                double cn = fg * c[bb * H + j] + ig * gg;
                c[bb * H + j] = cn;
                m[bb * H + j] = og * tanh(cn);
                if (gates) {
                    double *gt = gates + (t * B + bb) * G;
                    gt[j] = ig; gt[H + j] = fg; gt[2 * H + j] = gg; gt[3 * H + j] = og;
                }
                if (cs) cs[(t * B + bb) * H + j] = cn;
                if (ms) ms[(t * B + bb) * H + j] = m[bb * H + j];
            }

        /* h_t = m_t, or the projection P m_t */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long p = 0; p < Hr; ++p) {
                double v;
                if (Hp) {
                    v = 0.0;
                    for (long j = 0; j < H; ++j) v += P[p * H + j] * m[bb * H + j];
                } else {
                    v = m[bb * H + p];
                }
                yt[bb * Hr + p] = v;
            }
        memcpy(hp, yt, sizeof(double) * (size_t)B * Hr);
    }
    if (hT) memcpy(hT, hp, sizeof(double) * (size_t)B * Hr);
    if (cT) memcpy(cT, c, sizeof(double) * (size_t)B * H);
    free(z); free(m); free(c); free(hp);
    return 0;
}

/*
 * Backward pass.  Recomputes the forward states itself, then walks the
 * visited steps in reverse.  dhT[B][Hr] / dcT[B][H] NULL mean zeros.
 * Outputs (each may be NULL when not wanted): dx[T][B][I], dh0[B][Hr],
 * dc0[B][H], dW[4H][I], dR[4H][Hr], db[4H], dP[Hp][H].  Weight gradients are
 * overwritten (summed over time and batch).
 */
int lstm_oracle_backward(int T, int B, int I, int H, int Hp, int reverse,
                         const double *x, const double *h0, const double *c0,
                         const double *W, const double *R, const double *b, const double *P,
                         const double *dy, const double *dhT, const double *dcT,
                         double *dx, double *dh0, double *dc0,
                         double *dW, double *dR, double *db, double *dP)
{
    if (T < 1 || B < 1 || I < 1 || H < 1 || Hp < 0 || (Hp > 0 && !P))
        return -1;
    const long Hr = Hp ? Hp : H;
    const long G = 4L * H;
    double *y = malloc(sizeof(double) * (size_t)T * B * Hr);
    double *gates = malloc(sizeof(double) * (size_t)T * B * G);
    double *cs = malloc(sizeof(double) * (size_t)T * B * H);
    double *ms = malloc(sizeof(double) * (size_t)T * B * H);
    double *dz = malloc(sizeof(double) * (size_t)B * G);     /* gradient of z for this step */
    double *dh = malloc(sizeof(double) * (size_t)B * Hr);    /* gradient of h_t, all paths */
    double *dm = malloc(sizeof(double) * (size_t)B * H);     /* gradient of m_t */
    double *dhn = malloc(sizeof(double) * (size_t)B * Hr);   /* carried to h_{t-1} */
    double *dcn = malloc(sizeof(double) * (size_t)B * H);    /* carried to c_{t-1} */
    double *zeros_h = calloc((size_t)B * Hr, sizeof(double));
    double *zeros_c = calloc((size_t)B * H, sizeof(double));
    int rc = -1;
    if (!y || !gates || !cs || !ms || !dz || !dh || !dm || !dhn || !dcn || !zeros_h || !zeros_c)
        goto done;
    if (lstm_oracle_forward(T, B, I, H, Hp, reverse, x, h0, c0, W, R, b, P, y, NULL, NULL, gates, cs, ms))
        goto done;

    for (long i = 0; i < (long)B * Hr; ++i) dhn[i] = dhT ? dhT[i] : 0.0;
    for (long i = 0; i < (long)B * H; ++i) dcn[i] = dcT ? dcT[i] : 0.0;
    if (dW) memset(dW, 0, sizeof(double) * (size_t)G * I);
    if (dR) memset(dR, 0, sizeof(double) * (size_t)G * Hr);
    if (db) memset(db, 0, sizeof(double) * (size_t)G);
    if (dP) memset(dP, 0, sizeof(double) * (size_t)Hp * H);

    for (int s = T - 1; s >= 0; --s) {
        const long t = step_time(s, T, reverse);
        const long tp = reverse ? t + 1 : t - 1;          /* time of the previous visited step */
        const double *xt = x + t * B * I;
        const double *hprev = s ? y + tp * B * Hr : (h0 ? h0 : zeros_h);
        const double *cprev = s ? cs + tp * B * H : (c0 ? c0 : zeros_c);
        const double *gt = gates + t * B * G;
        const double *ct = cs + t * B * H;
        const double *mt = ms + t * B * H;

        /* dL/dh_t: the output's own gradient plus what flows back from t+1 */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long p = 0; p < Hr; ++p)
                dh[bb * Hr + p] = dy[(t * B + bb) * Hr + p] + dhn[bb * Hr + p];

        /* through the projection: dm = P^T dh (identity for a plain LSTM) */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long j = 0; j < H; ++j) {
                double v;
                if (Hp) {
                    v = 0.0;
                    for (long p = 0; p < Hp; ++p) v += P[p * H + j] * dh[bb * Hr + p];
                } else {
                    v = dh[bb * Hr + j];
                }
                dm[bb * H + j] = v;
            }

        /* through m = o tanh(c), c = f c_prev + i g and the gate non-linearities */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long j = 0; j < H; ++j) {
                const double *g4 = gt + bb * G;
                double ig = g4[j], fg = g4[H + j], gg = g4[2 * H + j], og = g4[3 * H + j];
                double tc = tanh(ct[bb * H + j]);
                double dmv = dm[bb * H + j];
                double d_o = dmv * tc;
                double d_c = dcn[bb * H + j] + dmv * og * (1.0 - tc * tc);
                double d_i = d_c * gg;
                double d_g = d_c * ig;
                double d_f = d_c * cprev[bb * H + j];
                double *dzb = dz + bb * G;
                dzb[j] = d_i * ig * (1.0 - ig);
                dzb[H + j] = d_f * fg * (1.0 - fg);
                dzb[2 * H + j] = d_g * (1.0 - gg * gg);
                dzb[3 * H + j] = d_o * og * (1.0 - og);
                dcn[bb * H + j] = d_c * fg;
            }

        /* input gradient dx_t = W^T dz and the carry dh_{t-1} = R^T dz */
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long k = 0; k < I; ++k) {
                double acc = 0.0;
                for (long r = 0; r < G; ++r) acc += W[r * I + k] * dz[bb * G + r];
                if (dx) dx[(t * B + bb) * I + k] = acc;
            }
#pragma omp parallel for collapse(2) schedule(static)
        for (long bb = 0; bb < B; ++bb)
            for (long k = 0; k < Hr; ++k) {
                double acc = 0.0;
                for (long r = 0; r < G; ++r) acc += R[r * Hr + k] * dz[bb * G + r];
                dhn[bb * Hr + k] = acc;
            }

        /* weight gradients, summed over the batch and accumulated over time */
#pragma omp parallel for schedule(static)
        for (long r = 0; r < G; ++r) {
            for (long bb = 0; bb < B; ++bb) {
                double d = dz[bb * G + r];
                if (dW)
                    for (long k = 0; k < I; ++k) dW[r * I + k] += d * xt[bb * I + k];
                if (dR)
                    for (long k = 0; k < Hr; ++k) dR[r * Hr + k] += d * hprev[bb * Hr + k];
                if (db) db[r] += d;
            }
        }
        if (Hp && dP) {
#pragma omp parallel for schedule(static)
            for (long p = 0; p < Hp; ++p)
                for (long bb = 0; bb < B; ++bb) {
                    double d = dh[bb * Hr + p];
                    for (long j = 0; j < H; ++j) dP[p * H + j] += d * mt[bb * H + j];
                }
        }
    }
    if (dh0) memcpy(dh0, dhn, sizeof(double) * (size_t)B * Hr);
    if (dc0) memcpy(dc0, dcn, sizeof(double) * (size_t)B * H);
    rc = 0;
done:
    free(y); free(gates); free(cs); free(ms); free(dz); free(dh); free(dm);
    free(dhn); free(dcn); free(zeros_h); free(zeros_c);
    return rc;
}
