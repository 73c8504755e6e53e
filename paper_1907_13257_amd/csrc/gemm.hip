// gemm.hip -- time-parallel matrix products of the LSTM step on gfx950
// matrix cores: the input projection X W^T + b for all T steps at once, and
// the gradients dX = dZ W, dW = dZ^T X, dR = dZ^T H_prev, dP = dH^T M.
//
// One kernel template covers all of them.  A workgroup (4 waves, 2x2) owns a
// BM x BN tile of C and walks K in stages of 64 bytes per row.  Both operands
// are staged in LDS with k contiguous in every row, so the fragment reads
// are 16-byte ds_reads for either element type.  An operand whose k is not the
// contiguous dimension in memory (the transposed operands of the weight
// gradients) is loaded with 16-byte global reads along m and transposed in
// registers before the LDS write.  Two LDS stages: the global loads of stage
// s+1 are in flight while stage s feeds the MFMAs.
#include "device_common.hpp"
#include "kernels.hpp"

namespace lstm355 {

namespace {

constexpr int KB = 64;            // bytes of k per stage and row
constexpr int PITCH = KB + 16;    // LDS row pitch (16 B of padding against bank conflicts)

struct GemmArgs {
    int M, N, K;
    const char *A; long lda;     // in elements
    const char *B; long ldb;
    char *C; long ldc;
    const float *bias;
    int beta;
    int tiles_n, ntiles, per_xcd;
};

// Loads `NC` 16-byte vectors of one operand stage into registers.
//   KMAJ:  chunk c = tid + i*256: row = c / 4, k-vector = c % 4.
//   !KMAJ: thread owns one m-vector (E rows) and NC consecutive k rows.
template <typename TI, int ROWS, bool KMAJ>
struct OperandLoader {
    static constexpr int E = 16 / (int)sizeof(TI);
    static constexpr int KS = KB / (int)sizeof(TI);         // k per stage
    static constexpr int NC = ROWS / 64;                    // vectors per thread
    u32x4 v[NC];

    __device__ __forceinline__ void load(const char *base, long ld, int r0, int rows_total, int k0, int K, int tid)
    {
        if (KMAJ) {
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                int c = tid + i * 256;
                int row = c >> 2, kv = c & 3;
                int gr = r0 + row, gk = k0 + kv * E;
                v[i] = (gr < rows_total && gk < K)
                           ? ldg16(base + ((long)gr * ld + gk) * (long)sizeof(TI))
                           : zero16();
            }
        } else {
            constexpr int MV = ROWS / E;                 // m-vectors per stage
            int mv = tid % MV, kg = tid / MV;
            int gm = r0 + mv * E;
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                int gk = k0 + kg * NC + i;
                v[i] = (gm < rows_total && gk < K)
                           ? ldg16(base + ((long)gk * ld + gm) * (long)sizeof(TI))
                           : zero16();
            }
        }
    }

    __device__ __forceinline__ void store(char *lds, int tid) const
    {
        if (KMAJ) {
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                int c = tid + i * 256;
                int row = c >> 2, kv = c & 3;
                *reinterpret_cast<u32x4 *>(lds + row * PITCH + kv * 16) = v[i];
            }
        } else {
            constexpr int MV = ROWS / E;
            int mv = tid % MV, kg = tid / MV;
            // element e of vector i is A(m = mv*E + e, k = kg*NC + i)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                char *dst = lds + (mv * E + e) * PITCH + kg * NC * (int)sizeof(TI);
                if (sizeof(TI) == 2) {
                    unsigned w[NC / 2 > 0 ? NC / 2 : 1];
#pragma unroll
                    for (int p = 0; p < NC / 2; ++p) {
                        unsigned lo = v[2 * p][e >> 1], hi = v[2 * p + 1][e >> 1];
                        lo = (e & 1) ? (lo >> 16) : (lo & 0xffffu);
                        hi = (e & 1) ? (hi & 0xffff0000u) : (hi << 16);
                        w[p] = lo | hi;
                    }
                    if (NC == 2) {
                        *reinterpret_cast<unsigned *>(dst) = w[0];
                    } else if (NC == 4) {
                        *reinterpret_cast<u32x2 *>(dst) = u32x2{w[0], w[1]};
                    } else {
#pragma unroll
                        for (int p = 0; p < NC / 2; ++p) reinterpret_cast<unsigned *>(dst)[p] = w[p];
                    }
                } else {
#pragma unroll
                    for (int p = 0; p < NC; ++p) reinterpret_cast<unsigned *>(dst)[p] = v[p][e];
                }
            }
        }
    }
};

template <typename TI, typename TO, int BM, int BN, bool AK, bool BKM>
__global__ __launch_bounds__(256, 2) void gemm_kernel(GemmArgs g)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int KS = KB / (int)sizeof(TI);
    constexpr int STAGE = (BM + BN) * PITCH;
    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];

    // XCD-aware order: consecutive workgroups go to different XCDs, so give
    // each XCD a contiguous run of tiles (shared A rows stay in its L2).
    const int bid = blockIdx.x;
    const int tile = (bid & 7) * g.per_xcd + (bid >> 3);
    if (tile >= g.ntiles) return;
    const int tm = tile / g.tiles_n, tn = tile % g.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;

    OperandLoader<TI, BM, AK> la;
    OperandLoader<TI, BN, BKM> lb;

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int nst = (g.K + KS - 1) / KS;
    la.load(g.A, g.lda, m0, g.M, 0, g.K, tid);
    lb.load(g.B, g.ldb, n0, g.N, 0, g.K, tid);
    la.store(smem, tid);
    lb.store(smem + BM * PITCH, tid);
    __syncthreads();

    for (int st = 0; st < nst; ++st) {
        const char *sa = smem + (st & 1) * STAGE;
        const char *sb = sa + BM * PITCH;
        const bool more = st + 1 < nst;
        if (more) {
            la.load(g.A, g.lda, m0, g.M, (st + 1) * KS, g.K, tid);
            lb.load(g.B, g.ldb, n0, g.N, (st + 1) * KS, g.K, tid);
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            u32x4 fa[FM], fb[FN];
            const int off = s * 32 + (lane >> 5) * 16;
#pragma unroll
            for (int i = 0; i < FM; ++i)
                fa[i] = *reinterpret_cast<const u32x4 *>(sa + (wm * WM + i * 32 + (lane & 31)) * PITCH + off);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                fb[j] = *reinterpret_cast<const u32x4 *>(sb + (wn * WN + j * 32 + (lane & 31)) * PITCH + off);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) mfma32(acc[i][j], fa[i], fb[j], TI{});
        }
        if (more) {
            char *da = smem + ((st + 1) & 1) * STAGE;
            la.store(da, tid);
            lb.store(da + BM * PITCH, tid);
        }
        __syncthreads();
    }

    // epilogue: lane holds rows 8*(v/4) + 4*(lane/32) + v%4, column lane%32
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int col = n0 + wn * WN + j * 32 + (lane & 31);
            if (col >= g.N) continue;
            const float bv = g.bias ? g.bias[col] : 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row < g.M) {
                    TO *cp = reinterpret_cast<TO *>(g.C) + (long)row * g.ldc + col;
                    float r = acc[i][j][v] + bv;
                    if (g.beta) r += to_f32(*cp);
                    *cp = from_f32<TO>(r);
                }
            }
        }
}

template <typename TI, typename TO, int BM, int BN, bool AK, bool BKM>
hipError_t launch_gemm(const GemmDesc &d, hipStream_t s)
{
    GemmArgs g;
    g.M = d.M; g.N = d.N; g.K = d.K;
    g.A = static_cast<const char *>(d.A); g.lda = d.lda;
    g.B = static_cast<const char *>(d.B); g.ldb = d.ldb;
    g.C = static_cast<char *>(d.C); g.ldc = d.ldc;
    g.bias = d.bias; g.beta = d.beta;
    const int tiles_m = (d.M + BM - 1) / BM;
    g.tiles_n = (d.N + BN - 1) / BN;
    g.ntiles = tiles_m * g.tiles_n;
    g.per_xcd = (g.ntiles + 7) / 8;
    const int grid = g.per_xcd * 8;
    hipLaunchKernelGGL((gemm_kernel<TI, TO, BM, BN, AK, BKM>), dim3(grid), dim3(256), 0, s, g);
    return hipGetLastError();
}

template <typename TI, typename TO, bool AK, bool BKM>
hipError_t dispatch_tiles(const GemmDesc &d, hipStream_t s)
{
    // Large outputs take 256x128 tiles; otherwise 128x128 keeps more
    // workgroups in flight on the 256 CUs.
    const long t256 = (long)((d.M + 255) / 256) * ((d.N + 127) / 128);
    if (t256 >= 512)
        return launch_gemm<TI, TO, 256, 128, AK, BKM>(d, s);
    return launch_gemm<TI, TO, 128, 128, AK, BKM>(d, s);
}

template <typename TI>
hipError_t dispatch_layout(const GemmDesc &d, hipStream_t s)
{
    if (d.a_kmajor && d.b_kmajor)
        return d.out_f32 ? dispatch_tiles<TI, float, true, true>(d, s) : dispatch_tiles<TI, TI, true, true>(d, s);
    if (d.a_kmajor && !d.b_kmajor)
        return d.out_f32 ? dispatch_tiles<TI, float, true, false>(d, s) : dispatch_tiles<TI, TI, true, false>(d, s);
    if (!d.a_kmajor && !d.b_kmajor && d.out_f32)
        return dispatch_tiles<TI, float, false, false>(d, s);
    return hipErrorNotSupported;
}

}  // namespace

hipError_t gemm(const GemmDesc &d, hipStream_t s, int kclass)
{
    if (d.M <= 0 || d.N <= 0 || d.K <= 0) return hipSuccess;
    const double flops = 2.0 * d.M * d.N * (double)d.K;
    const double es = (double)dsize(d.in);
    const double bytes = es * ((double)d.M * d.K + (double)d.N * d.K) +
                         (d.out_f32 ? 4.0 : es) * (double)d.M * d.N * (d.beta ? 2.0 : 1.0);
    ProfScope ps(kclass, s, flops, bytes);
    return d.in == DType::BF16 ? dispatch_layout<bf16_t>(d, s) : dispatch_layout<float>(d, s);
}

}  // namespace lstm355
