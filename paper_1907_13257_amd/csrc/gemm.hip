// gemm.hip -- time-parallel matrix products of the LSTM step on gfx950
// matrix cores: the input projection X W^T + b for all T steps at once, and
// the gradients dX = dZ W, dW = dZ^T X, dR = dZ^T H_prev, dP = dH^T M.
//
// One kernel template covers all of them.  A workgroup (4 waves, 2x2) owns a
// BM x BN tile of C (up to 256x256: 128x128 per wave, accumulators in AGPRs)
// and walks K in stages of KB bytes per row.  Both operands are staged in LDS
// with k contiguous in every row, so every fragment read is a 16-byte
// ds_read.  An operand whose k is not the contiguous dimension in memory (the
// transposed operands of the weight gradients) is loaded with 16-byte global
// reads along m and transposed in registers before the LDS write.  Two LDS
// stages: the global loads of stage s+1 are in flight while stage s feeds
// v_mfma_f32_32x32x16_bf16 (fp32 inputs: v_mfma_f32_32x32x2f32).
//
// Small outputs (the weight gradients are 4H x I at most, K = T*B long) can
// be split along K over several workgroups; every split writes an fp32
// partial tile and a second kernel sums the splits in a fixed order, so the
// result does not depend on scheduling.
#include "device_common.hpp"
#include "kernels.hpp"
#include "side_job.hpp"

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>

namespace lstm355 {

namespace {

struct GemmArgs {
    int M, N, K;
    const char *A; long lda;     // in elements
    const char *B; long ldb;
    char *C; long ldc;
    const float *bias;
    int beta;
    int tiles_n, ntiles, per_xcd;
    int band;                    // tile columns per band of the tile order (tiles_n: row-major)
    int kchunk;                  // K per split (multiple of the stage depth)
    float *partial;              // split > 1: fp32 partials [split][M][N]
    // second column block (see GemmDesc)
    int N1;
    const char *B2, *B3;
    long ldb2, ldb3, b2_bytes, b3_bytes;
    int ylo, yhi, yoff, hlo, hlen;
    char *C2;
    long ldc2;
    SideJob side;
    // fused cell update (see GemmDesc)
    int cell_h;
    const float *cell_prev;
    float *cell_c, *cell_cT;
    bf16_t *cell_m;
    long cell_ldm;
    // batch (blockIdx.z selects the product)
    int nbatch;
    struct {
        const char *A, *B, *B2;
        char *C, *C2;
        const float *sum_src;
        float *sum_dst;
    } bt[4];
};

// Global -> register -> LDS staging of one operand for one K stage.
//   KMAJ:  16-byte vector c = tid + i*256 is row c / VPR, k-vector c % VPR.
//   !KMAJ: thread owns one m-vector (E rows) and NC consecutive k rows, and
//          transposes them in registers (element e of vector i is
//          operand(m = mv*E + e, k = kg*NC + i)).
template <typename TI, int ROWS, bool KMAJ, int KB>
struct Loader {
    static constexpr int E = 16 / (int)sizeof(TI);
    static constexpr int KS = KB / (int)sizeof(TI);   // k per stage
    static constexpr int VPR = KB / 16;               // vectors per row per stage
    static constexpr int NC = ROWS * VPR / 256;       // vectors per thread
    static constexpr int PITCH = KB + 16;
    static constexpr int MV = ROWS / E;
    u32x4 v[NC];

    __device__ __forceinline__ void load(const char *base, long ld, int r0, int rows_total, int k0, int kend, int tid)
    {
        if (KMAJ) {
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                const int c = tid + i * 256;
                const int row = c / VPR, kv = c % VPR;
                const int gr = r0 + row, gk = k0 + kv * E;
                v[i] = (gr < rows_total && gk < kend) ? ldg16(base + ((long)gr * ld + gk) * (long)sizeof(TI))
                                                      : zero16();
            }
        } else {
            const int mv = tid % MV, kg = tid / MV;
            const int gm = r0 + mv * E;
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                const int gk = k0 + kg * NC + i;
                v[i] = (gm < rows_total && gk < kend) ? ldg16(base + ((long)gk * ld + gm) * (long)sizeof(TI))
                                                      : zero16();
            }
        }
    }

    __device__ __forceinline__ void store(char *lds, int tid) const
    {
        if (KMAJ) {
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                const int c = tid + i * 256;
                const int row = c / VPR, kv = c % VPR;
                *reinterpret_cast<u32x4 *>(lds + row * PITCH + kv * 16) = v[i];
            }
        } else {
            const int mv = tid % MV, kg = tid / MV;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                char *dst = lds + (mv * E + e) * PITCH + kg * NC * (int)sizeof(TI);
                if (sizeof(TI) == 2) {
                    unsigned w[NC / 2];
#pragma unroll
                    for (int p = 0; p < NC / 2; ++p) {
                        unsigned lo = v[2 * p][e >> 1], hi = v[2 * p + 1][e >> 1];
                        lo = (e & 1) ? (lo >> 16) : (lo & 0xffffu);
                        hi = (e & 1) ? (hi & 0xffff0000u) : (hi << 16);
                        w[p] = lo | hi;
                    }
                    if (NC == 8) {
                        *reinterpret_cast<u32x4 *>(dst) = u32x4{w[0], w[1], w[2], w[3]};
                    } else if (NC == 4) {
                        *reinterpret_cast<u32x2 *>(dst) = u32x2{w[0], w[1]};
                    } else {
#pragma unroll
                        for (int p = 0; p < NC / 2; ++p) reinterpret_cast<unsigned *>(dst)[p] = w[p];
                    }
                } else {
                    if (NC % 4 == 0) {
#pragma unroll
                        for (int p = 0; p < NC; p += 4)
                            *reinterpret_cast<u32x4 *>(dst + p * 4) = u32x4{v[p][e], v[p + 1][e], v[p + 2][e], v[p + 3][e]};
                    } else {
#pragma unroll
                        for (int p = 0; p < NC; ++p) reinterpret_cast<unsigned *>(dst)[p] = v[p][e];
                    }
                }
            }
        }
    }
};

template <typename TI, typename TO, int BM, int BN, int KB, bool AK, bool BKM>
__global__ __launch_bounds__(256, (BM * BN > 128 * 128) ? 1 : 2) void gemm_kernel(GemmArgs g)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int KS = KB / (int)sizeof(TI);
    constexpr int PITCH = KB + 16;
    constexpr int STAGE = (BM + BN) * PITCH;
    constexpr int SUB = KB / 32;                      // 32-byte k substeps per stage
    extern __shared__ __attribute__((aligned(16))) char smem[];

    // XCD-aware order: consecutive workgroups go to different XCDs, so give
    // each XCD a contiguous run of tiles (shared operand rows stay in its L2).
    const int bid = blockIdx.x;
    const int tile = (bid & 7) * g.per_xcd + (bid >> 3);
    if (tile >= g.ntiles) {
        run_side_job(g.side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
        return;
    }
    const int tm = tile / g.tiles_n, tn = tile % g.tiles_n;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = blockIdx.y * g.kchunk;
    const int kend = min(g.K, kbeg + g.kchunk);

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1;

    Loader<TI, BM, AK, KB> la;
    Loader<TI, BN, BKM, KB> lb;

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int nst = (kend - kbeg + KS - 1) / KS;
    if (nst > 0) {
        la.load(g.A, g.lda, m0, g.M, kbeg, kend, tid);
        lb.load(g.B, g.ldb, n0, g.N, kbeg, kend, tid);
        la.store(smem, tid);
        lb.store(smem + BM * PITCH, tid);
    }
    __syncthreads();

    for (int st = 0; st < nst; ++st) {
        const char *sa = smem + (st & 1) * STAGE;
        const char *sb = sa + BM * PITCH;
        const bool more = st + 1 < nst;
        if (more) {
            la.load(g.A, g.lda, m0, g.M, kbeg + (st + 1) * KS, kend, tid);
            lb.load(g.B, g.ldb, n0, g.N, kbeg + (st + 1) * KS, kend, tid);
        }
#pragma unroll
        for (int s = 0; s < SUB; ++s) {
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
    const bool split = g.partial != nullptr;
    float *part = split ? g.partial + (long)blockIdx.y * g.M * g.N : nullptr;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int col = n0 + wn * WN + j * 32 + (lane & 31);
            if (col >= g.N) continue;
            const float bv = (!split && g.bias) ? g.bias[col] : 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row < g.M) {
                    if (split) {
                        part[(long)row * g.N + col] = acc[i][j][v];
                    } else {
                        TO *cp = reinterpret_cast<TO *>(g.C) + (long)row * g.ldc + col;
                        float r = acc[i][j][v] + bv;
                        if (g.beta) r += to_f32(*cp);
                        *cp = from_f32<TO>(r);
                    }
                }
            }
        }
    run_side_job(g.side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
}

// ---------------------------------------------------------------------------
// bf16 kernel with direct global -> LDS loads (no register staging).
//
// Operands reach LDS through bounds-checked buffer loads that write LDS
// directly (16 bytes per lane; a wave fills 1 KiB per instruction).  Rows
// past the end of a K-major operand read as zero.  A ring of NS stages of KD
// k (KD = 32 or 64) keeps NS-1 stages of loads in flight while one is
// consumed.  LDS rows are XOR-swizzled in 16-byte chunks so that the lanes
// one LDS cycle serves (a 256-byte window of 64 four-byte banks) touch
// distinct chunk positions:
//   K-major tile [rows][2 KD bytes]: chunk c of row r lives at slot
//     c ^ ((r / RW) % CH), RW = 256 / (2 KD) rows per window, CH chunks per row;
//   M-major tile [KD k][rows]: chunk c of k-row k lives at slot c ^ (4 (k & 3)),
//     so the four k-rows read by 32 lanes of ds_read_b64_tr_b16 fall in
//     disjoint 64-byte ranges.
// M-major operands (the transposed operands of dW, dR, dP, dX) are read with
// ds_read_b64_tr_b16: in each group of 16 lanes, output lane i, element e is
// element (i % 4) of the 8 bytes addressed by source lane 4e + i/4, so source
// lanes addressing (k = kb + s/4, m = mb + 4 (s % 4)) deliver to lane i the
// four k values kb..kb+3 of column m = mb + i.
// ---------------------------------------------------------------------------
template <int ROWS, bool KMAJ, int KD, int NW>
struct DlLayout {
    static constexpr int RB = KD * 2;             // K-major: bytes per row per stage
    static constexpr int CH = RB / 16;            // K-major: chunks per row
    static constexpr int RW = 256 / RB;           // K-major: rows per 256-byte window
    static constexpr int RP = ROWS * 2;           // M-major: bytes per k-row
    static constexpr int BYTES = ROWS * RB;       // either layout
    static constexpr int NI = BYTES / 1024 / NW;  // 1 KiB instructions per wave per stage
    static_assert(NI * 1024 * NW == BYTES, "a stage must split evenly over the waves");

    __device__ static __forceinline__ int kslot(int row, int c) { return c ^ ((row / RW) % CH); }
    __device__ static __forceinline__ int mslot(int k, int c) { return c ^ (4 * (k & 3)); }
};

// One operand of one stage: ROWS rows, KD k, loaded by NW waves.
template <int ROWS, bool KMAJ, int KD, int NW>
struct DmaOperand {
    using L = DlLayout<ROWS, KMAJ, KD, NW>;
    u32x4 rsrc;                                   // buffer descriptor (base, limit, format)
    long ld;                                      // elements
    int r0;
    int ilv = 0;                                  // > 0 (K-major only): tile row n reads memory row
                                                  // (n % 4) * ilv + n / 4 (cell-major gate order)

    __device__ __forceinline__ void init(const char *base, long ld_, int r0_, long bound_bytes)
    {
        rsrc = buffer_desc(base, bound_bytes);
        ld = ld_;
        r0 = r0_;
    }

    __device__ __forceinline__ void issue(unsigned dst, int k0, int wave, int lane) const
    {
#pragma unroll
        for (int i = 0; i < L::NI; ++i) {
            const int q = wave * L::NI + i;
            const int byte = q * 1024 + lane * 16;
            unsigned off;
            if (KMAJ) {
                const int row = byte / L::RB, p = (byte % L::RB) >> 4;
                const int c = L::kslot(row, p);   // the swizzle is an involution
                const int n = r0 + row;
                const long mrow = ilv ? (long)(n & 3) * ilv + (n >> 2) : (long)n;
                off = (unsigned)(((mrow * ld + k0) << 1) + c * 16);
            } else {
                const int k = byte / L::RP, p = (byte % L::RP) >> 4;
                const int c = L::mslot(k, p);
                off = (unsigned)((((long)(k0 + k) * ld + r0) << 1) + c * 16);
            }
            dma16(rsrc, __builtin_amdgcn_readfirstlane(dst + q * 1024), off);
        }
    }
};

// Byte offset (within a stage's operand region) of this lane's fragment read
// for k substep s (16 k): K-major one b128; M-major two b64 transpose reads.
template <int ROWS, bool KMAJ, int KD>
__device__ __forceinline__ unsigned frag_off(int rowbase, int s, int r, int lane)
{
    using L = DlLayout<ROWS, KMAJ, KD, 1>;
    if (KMAJ) {
        const int row = rowbase + (lane & 31);
        const int c = 2 * s + (lane >> 5);
        return (unsigned)(row * L::RB + (L::kslot(row, c) << 4));
    } else {
        const int gq = lane >> 4, sl = lane & 15;
        const int k = 16 * s + (gq >> 1) * 8 + 4 * r + (sl >> 2);
        const int m = rowbase + 16 * (gq & 1) + 4 * (sl & 3);
        const int c = m >> 3;
        return (unsigned)(k * L::RP + (L::mslot(k, c) << 4) + ((m & 7) << 1));
    }
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4 lds_u32x4_t;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

template <int F, int ROWS, bool KMAJ, int KD>
__device__ __forceinline__ void read_frags(u32x4 (&f)[F], const char *base, int rowbase0, int s, int lane)
{
#pragma unroll
    for (int i = 0; i < F; ++i) {
        if (KMAJ) {
            f[i] = *(const lds_u32x4_t *)(base + frag_off<ROWS, true, KD>(rowbase0 + i * 32, s, 0, lane));
        } else {
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_s16x4_t *)(base + frag_off<ROWS, false, KD>(rowbase0 + i * 32, s, 0, lane)));
            const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_s16x4_t *)(base + frag_off<ROWS, false, KD>(rowbase0 + i * 32, s, 1, lane)));
            const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
            f[i] = u32x4{l2[0], l2[1], h2[0], h2[1]};
        }
    }
}

// Four consecutive values of a row of C: one 16-byte fp32 store, or one
// 8-byte store of four 16-bit values.
template <typename TO>
__device__ __forceinline__ void store4(TO *p, f32x4 v);
template <>
__device__ __forceinline__ void store4<float>(float *p, f32x4 v)
{
    *reinterpret_cast<f32x4 *>(p) = v;
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t *p, f32x4 v)
{
    const unsigned lo = (unsigned)f32_to_bf16(v[0]) | ((unsigned)f32_to_bf16(v[1]) << 16);
    const unsigned hi = (unsigned)f32_to_bf16(v[2]) | ((unsigned)f32_to_bf16(v[3]) << 16);
    *reinterpret_cast<u32x2 *>(p) = u32x2{lo, hi};
}

template <>
__device__ __forceinline__ void store4<f16_t>(f16_t *p, f32x4 v)
{
    typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
    *reinterpret_cast<f16x4 *>(p) =
        f16x4{f32_to_f16_sat(v[0]), f32_to_f16_sat(v[1]), f32_to_f16_sat(v[2]), f32_to_f16_sat(v[3])};
}

__device__ __forceinline__ void wait_lds_only() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Tile order: bands of g.band tile columns, each band row-major.  The XCD
// groups take consecutive ranges of this order, so a group's tiles cover a
// roughly square block of C and share both operands' rows in its L2 (the
// host picks the band width that minimises the operand bytes per group).
__device__ __forceinline__ void tile_of(const GemmArgs &g, int lin, int &tm, int &tn)
{
    const int tiles_m = g.ntiles / g.tiles_n;
    const int full = g.tiles_n / g.band;
    const int per_band = tiles_m * g.band;
    const int b = lin / per_band;
    if (b < full) {
        const int r = lin - b * per_band;
        tm = r / g.band;
        tn = b * g.band + r % g.band;
    } else {   // the narrower last band
        const int r = lin - full * per_band, wl = g.tiles_n - full * g.band;
        tm = r / wl;
        tn = full * g.band + r % wl;
    }
}

// NWM x NWN waves; wave (wm, wn) owns the (BM/NWM) x (BN/NWN) block of the tile.
// CB: the instantiation used when C is accumulated into (beta = 1, no split).
// GT: fused cell update (GemmDesc::cell_h): tile columns are cell-major gates
// (column n is gate n % 4 of cell n / 4), and the epilogue applies the cell
// equations to the four gates of each (row, cell) through LDS.
// Four-wave configurations whose stages leave room for two workgroups per CU
// are compiled for two (at most 256 registers per wave, accumulators and
// operands together); otherwise the compiler may spend up to 512 and a CU
// then holds one workgroup, one wave per SIMD.
template <int BM, int BN, int KD, int NS, int NW>
constexpr int dl_min_blocks()
{
    return (NW == 4 && NS * (BM + BN) * KD * 2 <= 80 * 1024) ? 2 : 1;
}

template <typename TO, int BM, int BN, bool AK, bool BKM, int KD, int NS, int NWM, int NWN, bool CB = false,
          bool GT = false>
__global__ __launch_bounds__(64 * NWM * NWN, (dl_min_blocks<BM, BN, KD, NS, NWM * NWN>()))
void gemm_dl_kernel(GemmArgs g)
{
    if (g.nbatch > 1) {   // product blockIdx.z of a batch (product 0's pointers are g's own)
        // constant indices keep the arguments in scalar registers
        const int z = blockIdx.z;
#pragma unroll
        for (int b = 1; b < 4; ++b)
            if (z == b) {
                g.A = g.bt[b].A; g.B = g.bt[b].B; g.B2 = g.bt[b].B2;
                g.C = g.bt[b].C; g.C2 = g.bt[b].C2;
                g.side.sum_src = g.bt[b].sum_src; g.side.sum_dst = g.bt[b].sum_dst;
            }
    }
    static_assert(!GT || (CB && BKM && BN % 4 == 0), "the cell update accumulates onto C with a k-major B");
    constexpr int NW = NWM * NWN;
    constexpr int WM = BM / NWM, WN = BN / NWN;
    constexpr int FM = WM / 32, FN = WN / 32;
    static_assert(FM * 32 * NWM == BM && FN * 32 * NWN == BN, "wave tiles are multiples of 32");
    using LA = DlLayout<BM, AK, KD, NW>;
    using LB = DlLayout<BN, BKM, KD, NW>;
    constexpr int ABYTES = LA::BYTES, STAGE = LA::BYTES + LB::BYTES;
    constexpr int LPW = LA::NI + LB::NI;          // DMA instructions per wave per stage
    extern __shared__ __attribute__((aligned(1024))) char smem[];

    const int bid = blockIdx.x;
    const int tile = (bid & 7) * g.per_xcd + (bid >> 3);
    if (tile >= g.ntiles) {
        run_side_job(g.side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
        return;
    }
    int tm, tn;
    tile_of(g, tile, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    // second column block: its own B operand segments, k range and output
    constexpr bool DUAL_OK = !AK && !BKM;
    const bool second = DUAL_OK && g.N1 > 0 && n0 >= g.N1;
    int kbeg = blockIdx.y * g.kchunk;
    int kend = min(g.K, kbeg + g.kchunk);
    if (second && !g.B3) {   // no h0 segment: only the B2 range contributes
        kbeg = g.ylo;
        kend = g.yhi;
    }
    // a last partial stage only when both operands are m-major: its rows past
    // K lie beyond the operands' buffer bounds and load as zeros
    const int nst = (kend - kbeg + KD - 1) / KD;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % NWM, wn = wave / NWM;

    DmaOperand<BM, AK, KD, NW> da;
    DmaOperand<BN, BKM, KD, NW> db;    // B, or B2 for the second block
    DmaOperand<BN, BKM, KD, NW> dh;    // B3 (second block only)
    // (second block without an h0 segment: rows of A past its k range read
    // zero, so a last stage that reaches past it adds nothing)
    da.init(g.A, g.lda, m0, AK ? (long)g.M * g.lda * 2 : (long)(second && !g.B3 ? g.yhi : g.K) * g.lda * 2);
    if (!second) {
        db.init(g.B, g.ldb, n0, BKM ? (long)g.N * g.ldb * 2 : (long)g.K * g.ldb * 2);
        if (GT) db.ilv = g.cell_h;
    } else {
        db.init(g.B2, g.ldb2, n0 - g.N1, g.b2_bytes);
        dh.init(g.B3 ? g.B3 : g.B2, g.ldb3, n0 - g.N1, g.B3 ? g.b3_bytes : 0);
    }
    auto issue_b = [&](unsigned dst, int k0) {
        if (!second)
            db.issue(dst, k0, wave, lane);
        else if (k0 >= g.hlo && k0 < g.hlo + g.hlen)
            dh.issue(dst, k0 - g.hlo, wave, lane);
        else
            db.issue(dst, k0 + g.yoff, wave, lane);
    };

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // Fused cell update: the C tile (the input projection, read through the
    // cell-major column remap) and the previous cell state do not depend on
    // the product, so they are loaded before the main loop and their latency
    // overlaps it.  The loads are older than stage 0's, so the first stage
    // wait covers them too.
    constexpr int CELLS_T = BN / 4;
    constexpr int NQ = GT ? (BM * CELLS_T) / (64 * NW) : 1;   // (row, cell) pairs per thread
    static_assert(!GT || NQ * 64 * NW == BM * CELLS_T, "the cell pairs split evenly over the threads");
    float cpre[GT ? FM : 1][GT ? FN : 1][16];
    float cprev_pre[NQ];
    if constexpr (GT) {
        const float *cg = reinterpret_cast<const float *>(g.C);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int col = n0 + wn * WN + j * 32 + (lane & 31);
                const long cc = (long)(col & 3) * g.cell_h + (col >> 2);
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = m0 + wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                    cpre[i][j][v] = (row < g.M && col < g.N) ? cg[(long)row * g.ldc + cc] : 0.0f;
                }
            }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int p = tid + q * 64 * NW, row = m0 + p / CELLS_T, cell = n0 / 4 + p % CELLS_T;
            cprev_pre[q] = (g.cell_prev && row < g.M && cell < g.cell_h) ? g.cell_prev[(long)row * g.cell_h + cell]
                                                                         : 0.0f;
        }
    }

    const unsigned sbase = lds_addr(smem);
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < nst) {
            const unsigned st_base = sbase + s * STAGE;
            da.issue(st_base, kbeg + s * KD, wave, lane);
            issue_b(st_base + ABYTES, kbeg + s * KD);
        }

    for (int st = 0; st < nst; ++st) {
        // stage st has landed once at most the later stages' loads are outstanding
        if (st + NS - 2 < nst)
            waitcnt_vm<(NS - 2) * LPW>();
        else
            waitcnt_vm<0>();
        asm volatile("s_barrier" ::: "memory");
        if (st + NS - 1 < nst) {
            const unsigned st_base = sbase + ((st + NS - 1) % NS) * STAGE;
            da.issue(st_base, kbeg + (st + NS - 1) * KD, wave, lane);
            issue_b(st_base + ABYTES, kbeg + (st + NS - 1) * KD);
        }
        const char *abase = smem + (st % NS) * STAGE;
        const char *bbase = abase + ABYTES;
        // raised wave priority while the stage's products issue: the
        // arbiter then favours waves with matrix work over waves issuing
        // loads or waiting at the barrier ([dW | dR] at 4096 x 2048 x 6400:
        // 128.7 -> 122.8 us, the other products unchanged)
        __builtin_amdgcn_s_setprio(3);
#pragma unroll
        for (int s = 0; s < KD / 16; ++s) {
            u32x4 fa[FM], fb[FN];
            read_frags<FM, BM, AK, KD>(fa, abase, wm * WM, s, lane);
            read_frags<FN, BN, BKM, KD>(fb, bbase, wn * WN, s, lane);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) mfma32(acc[i][j], fa[i], fb[j], bf16_t{});
        }
        __builtin_amdgcn_s_setprio(0);
    }

    const bool split = g.partial != nullptr;
    float *part = split ? g.partial + (long)blockIdx.y * g.M * g.N : nullptr;
    TO *cbase = reinterpret_cast<TO *>(second ? g.C2 : g.C);
    const long ldc = second ? g.ldc2 : g.ldc;
    const int coff = second ? g.N1 : 0;
    // column of C (the gate pre-activations) that tile column `col` holds
    auto ccol = [&](int col) -> long { return GT ? (long)(col & 3) * g.cell_h + (col >> 2) : (long)(col - coff); };
    // beta, CB instantiations: C is read block by block before anything is
    // stored (a load may not pass an earlier store to C in program order, so
    // interleaving them would expose one memory latency per element).  The
    // other instantiations add C element by element: the staging registers
    // would lower their occupancy.
    constexpr bool CPRE = CB;
    if constexpr (GT) {   // C was loaded before the main loop
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] += cpre[i][j][v];
    } else if (CPRE && !split && g.beta) {
        constexpr int CJ = 1;   // one 32x32 block (16 values) per batch of loads
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j0 = 0; j0 < FN; j0 += CJ) {
                float cv[CJ][16];
#pragma unroll
                for (int j = 0; j < CJ; ++j) {
                    const int col = n0 + wn * WN + (j0 + j) * 32 + (lane & 31);
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int row = m0 + wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                        cv[j][v] = (row < g.M && col < g.N) ? to_f32(cbase[(long)row * ldc + ccol(col)]) : 0.0f;
                    }
                }
#pragma unroll
                for (int j = 0; j < CJ; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[i][j0 + j][v] += cv[j][v];
            }
    }
    if constexpr (GT) {
        // z of the tile into LDS (the operand stages are no longer read), then
        // one (row, cell) pair per thread and pass: the four gates of a cell
        // are adjacent columns
        constexpr int ZP = BN + 4;
        static_assert(BM * ZP * 4 <= NS * STAGE, "the z tile fits in the operand stages");
        float *zt = reinterpret_cast<float *>(smem);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int r = wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                    zt[r * ZP + wn * WN + j * 32 + (lane & 31)] = acc[i][j][v];
                }
        __syncthreads();
        const int H = g.cell_h;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int p = tid + q * 64 * NW;
            const int r = p / CELLS_T, u = p % CELLS_T;
            const int row = m0 + r, cell = n0 / 4 + u;
            if (row >= g.M || cell >= H) continue;
            const f32x4 z = *reinterpret_cast<const f32x4 *>(&zt[r * ZP + 4 * u]);
            const float ig = sigmoid_f(z[0]), fg = sigmoid_f(z[1]), gg = tanh_f(z[2]), og = sigmoid_f(z[3]);
            const long e = (long)row * H + cell;
            const float c = fg * cprev_pre[q] + ig * gg;
            float *gp = reinterpret_cast<float *>(cbase) + (long)row * ldc + cell;
            gp[0] = ig;
            gp[H] = fg;
            gp[2 * H] = gg;
            gp[3 * H] = og;
            g.cell_c[e] = c;
            g.cell_m[(long)row * g.cell_ldm + cell] = f32_to_bf16(og * tanh_f(c));
            if (g.cell_cT) g.cell_cT[e] = c;
        }
        run_side_job(g.side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
        return;
    }
    // Plain stores (no accumulation into C, four-column aligned C) and split
    // partials: each 32x32 block goes through the wave's own LDS scratch so
    // that every lane stores four consecutive columns of a row at once (16
    // bytes fp32, 8 bytes 16-bit) instead of one element per block row: a
    // quarter of the store instructions, which bound the epilogue more than
    // its bytes do.
    constexpr int SP = 36;                        // scratch row pitch (floats): 16-byte rows, few bank conflicts
    static_assert(NW * 32 * SP * 4 <= NS * STAGE, "the epilogue scratch fits in the operand stages");
    const bool vec_out =
        split ? (g.N % 4) == 0 && (reinterpret_cast<uintptr_t>(part) & 15) == 0
              : !g.beta && (g.N % 4) == 0 && (ldc % 4) == 0 && (coff % 4) == 0 &&
                    (reinterpret_cast<uintptr_t>(cbase) & (4 * sizeof(TO) - 1)) == 0;
    if (vec_out) {
        float *scr = reinterpret_cast<float *>(smem) + wave * 32 * SP;
        __syncthreads();   // every wave has finished reading the operand stages
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                // lane holds column lane % 32 of rows 8 (v / 4) + 4 (lane / 32) + v % 4
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    scr[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * SP + (lane & 31)] = acc[i][j][v];
                wait_lds_only();
                // read back row-major: four consecutive columns per lane and pass
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int q = r * 64 + lane, rr = q >> 3, c4 = (q & 7) * 4;
                    const f32x4 x4 = *reinterpret_cast<const f32x4 *>(&scr[rr * SP + c4]);
                    const int row = m0 + wm * WM + i * 32 + rr, col = n0 + wn * WN + j * 32 + c4;
                    if (row < g.M && col < g.N) {
                        if (split) {
                            store4<float>(part + (long)row * g.N + col, x4);
                        } else {
                            f32x4 o = x4;
                            if (g.bias) {
                                const f32x4 b4 = *reinterpret_cast<const f32x4 *>(&g.bias[col]);
                                o = o + b4;
                            }
                            store4<TO>(cbase + (long)row * ldc + (col - coff), o);
                        }
                    }
                }
                wait_lds_only();   // the reads are done before the next block overwrites the scratch
            }
        run_side_job(g.side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
        return;
    }
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int col = n0 + wn * WN + j * 32 + (lane & 31);
            if (col >= g.N) continue;
            const float bv = (!split && g.bias) ? g.bias[col] : 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row < g.M) {
                    if (split) {
                        part[(long)row * g.N + col] = acc[i][j][v];
                    } else {
                        TO *cp = cbase + (long)row * ldc + (col - coff);
                        float r = acc[i][j][v] + bv;
                        if (!CPRE && g.beta) r += to_f32(*cp);
                        *cp = from_f32<TO>(r);
                    }
                }
            }
        }
    run_side_job(g.side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
}

// C[m][n] = (beta ? C : 0) + bias[n] + sum over splits of partial[s][m][n], in split order.
template <typename TO>
__global__ __launch_bounds__(256) void splitk_reduce(const float *__restrict__ partial, int splits, int M, int N,
                                                      const float *bias, int beta, TO *C, long ldc)
{
    const long total = (long)M * N;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
        const int m = (int)(i / N), n = (int)(i % N);
        float r = 0.0f;
        for (int s = 0; s < splits; ++s) r += partial[(long)s * total + i];
        if (bias) r += bias[n];
        TO *cp = C + (long)m * ldc + n;
        if (beta) r += to_f32(*cp);
        *cp = from_f32<TO>(r);
    }
}

// The same four columns at a time (N and ldc multiples of 4, C 16-byte
// aligned), with the split loop unrolled so that several partial loads are in
// flight per thread.
template <typename TO>
__global__ __launch_bounds__(256) void splitk_reduce4(const float *__restrict__ partial, int splits, int M, int N,
                                                       const float *bias, int beta, TO *C, long ldc)
{
    const long total = (long)M * N, total4 = total / 4;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < total4; i += (long)gridDim.x * 256) {
        const long e = i * 4;
        const int m = (int)(e / N), n = (int)(e % N);
        f32x4 r = {0.f, 0.f, 0.f, 0.f};
        int sp = 0;
        for (; sp + 4 <= splits; sp += 4) {
            const f32x4 a = *reinterpret_cast<const f32x4 *>(partial + (long)sp * total + e);
            const f32x4 b = *reinterpret_cast<const f32x4 *>(partial + (long)(sp + 1) * total + e);
            const f32x4 c = *reinterpret_cast<const f32x4 *>(partial + (long)(sp + 2) * total + e);
            const f32x4 d = *reinterpret_cast<const f32x4 *>(partial + (long)(sp + 3) * total + e);
#pragma unroll
            for (int v = 0; v < 4; ++v) r[v] = r[v] + a[v] + b[v] + c[v] + d[v];
        }
        for (; sp < splits; ++sp) {
            const f32x4 a = *reinterpret_cast<const f32x4 *>(partial + (long)sp * total + e);
#pragma unroll
            for (int v = 0; v < 4; ++v) r[v] += a[v];
        }
        TO *cp = C + (long)m * ldc + n;
        if (beta) {   // all four loads before the first store
            float c4[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) c4[v] = to_f32(cp[v]);
#pragma unroll
            for (int v = 0; v < 4; ++v) r[v] += c4[v];
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) cp[v] = from_f32<TO>(bias ? r[v] + bias[n + v] : r[v]);
    }
}

// Band width (tile columns) for the tile order: a group of `per_xcd` tiles
// arranged (per_xcd / w) x w reads about per_xcd/w * BM rows of A and w * BN
// rows of B; the power of two nearest sqrt(per_xcd * BM / BN) minimises the
// sum.  Bands are used only where they cut that sum by a third or more
// (BigLSTM's input projection: 5x; the headline layer's: 1.33x, where the
// changed cache contents slowed the next kernels by more than they saved).
// LSTM355_GEMM_BAND overrides (tests and tuning).
int band_width(int tiles_m, int tiles_n, int per_xcd, int BM, int BN)
{
    auto rows_read = [&](int w) {
        const int w_eff = w < tiles_n ? w : tiles_n;
        const double rows_of_a = std::min((double)tiles_m, std::ceil((double)per_xcd / w_eff)) * BM;
        return rows_of_a + (double)std::min(per_xcd, w_eff) * BN;
    };
    const char *env = std::getenv("LSTM355_GEMM_BAND");
    int w = 0;
    if (env) {
        w = std::atoi(env);
    } else {
        const double best = std::sqrt((double)per_xcd * BM / BN);
        w = 1;
        while (w * 2 <= tiles_n && (double)(w * 2) <= best * 1.4142) w *= 2;
        if (rows_read(tiles_n) < 1.5 * rows_read(w)) w = tiles_n;
    }
    if (w < 1 || w > tiles_n) w = tiles_n;
    return w;
}

template <typename TO>
hipError_t launch_splitk_reduce(const GemmDesc &d, int splits, hipStream_t s)
{
    const long total = (long)d.M * d.N;
    const bool vec = d.N % 4 == 0 && d.ldc % 4 == 0 && (reinterpret_cast<uintptr_t>(d.C) & 15) == 0;
    long grid = ((vec ? total / 4 : total) + 255) / 256;
    if (grid > 4096) grid = 4096;
    if (vec)
        hipLaunchKernelGGL(splitk_reduce4<TO>, dim3((unsigned)grid), dim3(256), 0, s, d.splitk_ws, splits, d.M, d.N,
                           d.bias, d.beta, reinterpret_cast<TO *>(d.C), d.ldc);
    else
        hipLaunchKernelGGL(splitk_reduce<TO>, dim3((unsigned)grid), dim3(256), 0, s, d.splitk_ws, splits, d.M, d.N,
                           d.bias, d.beta, reinterpret_cast<TO *>(d.C), d.ldc);
    return hipGetLastError();
}

template <typename TO, int BM, int BN, bool AK, bool BKM, int KD, int NS, int NWM, int NWN, bool CB = false,
          bool GT = false>
hipError_t launch_gemm_dl(const GemmDesc &d, int splits, hipStream_t s)
{
    constexpr int LDS = NS * (BM + BN) * KD * 2;
    GemmArgs g;
    if (d.nbatch > 1) splits = 1;   // batched products are never split
    g.M = d.M; g.N = d.N; g.K = d.K;
    g.A = static_cast<const char *>(d.A); g.lda = d.lda;
    g.B = static_cast<const char *>(d.B); g.ldb = d.ldb;
    g.C = static_cast<char *>(d.C); g.ldc = d.ldc;
    g.bias = d.bias; g.beta = d.beta;
    const int tiles_m = (d.M + BM - 1) / BM;
    g.tiles_n = (d.N + BN - 1) / BN;
    g.ntiles = tiles_m * g.tiles_n;
    g.per_xcd = (g.ntiles + 7) / 8;
    g.band = band_width(tiles_m, g.tiles_n, g.per_xcd, BM, BN);
    g.kchunk = ((d.K + splits - 1) / splits + KD - 1) / KD * KD;
    splits = (d.K + g.kchunk - 1) / g.kchunk;
    if (d.partials > 1 && splits != d.partials) return hipErrorInvalidValue;
    g.partial = splits > 1 ? d.splitk_ws : nullptr;
    g.N1 = d.N1;
    g.B2 = static_cast<const char *>(d.B2); g.ldb2 = d.ldb2; g.b2_bytes = d.b2_bytes;
    g.B3 = static_cast<const char *>(d.B3); g.ldb3 = d.ldb3; g.b3_bytes = d.b3_bytes;
    g.ylo = d.ylo; g.yhi = d.yhi; g.yoff = d.yoff; g.hlo = d.hlo; g.hlen = d.hlen;
    g.C2 = static_cast<char *>(d.C2); g.ldc2 = d.ldc2;
    g.side = d.side;
    g.cell_h = GT ? d.cell_h : 0;
    g.cell_prev = d.cell_prev; g.cell_c = d.cell_c; g.cell_cT = d.cell_cT;
    g.cell_m = static_cast<bf16_t *>(d.cell_m); g.cell_ldm = d.cell_ldm;
    auto kern = gemm_dl_kernel<TO, BM, BN, AK, BKM, KD, NS, NWM, NWN, CB, GT>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
    if (e != hipSuccess) return e;
    g.nbatch = 1;
    if (d.nbatch > 1) {
        if (d.nbatch > 4 || !d.batch) return hipErrorInvalidValue;
        g.nbatch = d.nbatch;
        for (int b = 0; b < d.nbatch; ++b) {
            const GemmDesc &e = d.batch[b];
            g.bt[b].A = static_cast<const char *>(e.A);
            g.bt[b].B = static_cast<const char *>(e.B);
            g.bt[b].B2 = static_cast<const char *>(e.B2);
            g.bt[b].C = static_cast<char *>(e.C);
            g.bt[b].C2 = static_cast<char *>(e.C2);
            g.bt[b].sum_src = e.side.sum_src;
            g.bt[b].sum_dst = e.side.sum_dst;
        }
    }
    hipLaunchKernelGGL(kern, dim3(g.per_xcd * 8, splits, g.nbatch), dim3(64 * NWM * NWN), LDS, s, g);
    e = hipGetLastError();
    if (e != hipSuccess || splits == 1 || d.partials > 1) return e;
    return launch_splitk_reduce<TO>(d, splits, s);
}

template <typename TI, typename TO, int BM, int BN, int KB, bool AK, bool BKM>
hipError_t launch_gemm(const GemmDesc &d, int splits, hipStream_t s)
{
    if (d.nbatch > 1) return hipErrorInvalidValue;   // batches run on the direct-to-LDS kernel only
    constexpr int KS = KB / (int)sizeof(TI);
    constexpr int LDS = 2 * (BM + BN) * (KB + 16);
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
    g.band = g.tiles_n;
    g.kchunk = ((d.K + splits - 1) / splits + KS - 1) / KS * KS;
    splits = (d.K + g.kchunk - 1) / g.kchunk;
    if (d.partials > 1 && splits != d.partials) return hipErrorInvalidValue;
    g.partial = splits > 1 ? d.splitk_ws : nullptr;
    g.N1 = 0; g.B2 = g.B3 = nullptr; g.C2 = nullptr;
    g.side = d.side;
    auto kern = gemm_kernel<TI, TO, BM, BN, KB, AK, BKM>;
    if (LDS > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(g.per_xcd * 8, splits), dim3(256), LDS, s, g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || splits == 1 || d.partials > 1) return e;
    return launch_splitk_reduce<TO>(d, splits, s);
}

// Tile and split choice: a crude model of per-CU efficiency per tile shape,
// quantised over 256 CUs, plus the traffic of the split-K partials.
struct Choice {
    int tile;     // 0: 256x256, 1: 256x128, 2: 128x256, 3: 128x128
    int splits;
};

// Tile configurations of the direct-to-LDS kernel (bf16):
//   index: BM x BN, waves (NWM x NWN), k per stage, ring stages
//   0: 256x256, 2x4, 32, 4      1: 256x128, 4x2, 32, 3    2: 128x256, 2x4, 32, 3
//   3: 128x128, 2x2, 32, 4      4: 256x256, 4x2, 32, 4    5: 128x128, 2x2, 64, 2
//   6: 256x128, 4x2, 64, 2      7: 128x256, 2x4, 64, 2    8: 256x256, 2x4, 64, 2
//   9: 256x256, 2x2, 32, 4     10: 256x256, 2x2, 64, 2   11: 128x256, 2x2, 32, 3
//  12: 256x128, 2x2, 32, 3     13: 128x256, 2x4, 64, 3   14: 256x128, 4x2, 64, 3
//  15: 128x128, 2x2, 64, 3     16: 128x128, 2x2, 64, 4   17: 128x128, 2x2, 32, 8
//  18: 64x128, 2x2, 64, 3       19: 64x64, 2x2, 64, 4     20: 128x64, 2x2, 64, 3
//  21: 256x256, 4x4, 32, 4     22: 256x256, 4x4, 64, 2   23: 256x128, 4x4, 64, 3
//  24: 128x256, 4x4, 64, 3
// (16 and 17 keep 96 / 112 KiB of operands in flight per workgroup: the
// per-step recurrent products stream their weights from HBM once; 18-20
// give the skinny per-step products more workgroups; 21-24 are one
// workgroup of 16 waves per CU, which loads a third fewer operand bytes per
// product than two 128x256 workgroups.  An operand whose rows
// are the contiguous dimension needs 128 of them per tile: its LDS swizzle
// spans 16 chunks of 16 bytes.)
constexpr int NTILES = 25;
const int kTileBM[NTILES] = {256, 256, 128, 128, 256, 128, 256, 128, 256, 256, 256, 128, 256,
                             128, 256, 128, 128, 128, 64,  64,  128, 256, 256, 256, 128};
const int kTileBN[NTILES] = {256, 128, 256, 128, 256, 128, 128, 256, 256, 256, 256, 256, 128,
                             256, 128, 128, 128, 128, 128, 64,  64,  256, 256, 128, 256};
const int kTileKD[NTILES] = {32, 32, 32, 32, 32, 64, 64, 64, 64, 32, 64, 32, 32,
                             64, 64, 64, 64, 32, 64, 64, 64, 32, 64, 64, 64};
// Workgroups of each configuration that fit on one CU (LDS-limited).
const int kTileSlots[NTILES] = {1, 1, 1, 2, 1, 2, 1, 1, 1, 1, 1, 2, 2, 1, 1, 1, 1, 1, 2, 2, 2, 1, 1, 1, 1};

bool dl_ok(const GemmDesc &d, int BM, int BN, int splits);
bool tile_fits(const GemmDesc &d, int t);
bool env_choice(Choice *c);

// Split count for tile shape BM x BN with `slots` workgroups per CU: enough
// k splits to fill the CUs, against the cost of the fp32 partials.
int model_splits(const GemmDesc &d, int BM, int BN, int slots, int kd)
{
    const double cu_rate = 4096.0 * 2.4e9 * 0.35;
    const long tiles = (long)((d.M + BM - 1) / BM) * ((d.N + BN - 1) / BN);
    int best = 1;
    double best_t = 1e30;
    for (int sp = 1; sp <= 64; sp *= 2) {
        if (sp > 1 && (!d.splitk_ws || (size_t)sp * d.M * d.N > d.splitk_ws_floats)) break;
        if (sp > 1 && d.K / sp < 4 * kd) break;
        const long items = tiles * sp;
        const long waves = (items + 256L * slots - 1) / (256L * slots);
        double tt = waves * 2.0 * BM * BN * ((double)d.K / sp) / (cu_rate / slots);
        if (sp > 1) tt += ((double)sp + 1.0) * d.M * d.N * 4.0 / 5.0e12 + 3e-6;
        if (tt < best_t * 0.97) {
            best_t = tt;
            best = sp;
        }
    }
    return best;
}

Choice choose(const GemmDesc &d, size_t es)
{
    static const int BMs[4] = {256, 256, 128, 128}, BNs[4] = {256, 128, 256, 128};
    static const double eff[4] = {1.0, 0.8, 0.8, 0.55};
    {
        Choice c;
        if (env_choice(&c)) {   // tuning override; a tile without a split count gets the modelled one
            if (c.splits == 0) c.splits = model_splits(d, kTileBM[c.tile], kTileBN[c.tile], kTileSlots[c.tile],
                                                       kTileKD[c.tile]);
            return c;
        }
    }
    if (es == 2 && d.M <= 256 && d.K % 64 == 0 && dl_ok(d, 128, 128, 1)) {
        // skinny products (one step of the stepwise recurrence) stream their
        // weight operand once.  Measured on the wide LSTMP layer's per-step
        // shapes (M = 128): accumulating with a k-contiguous weight, 128x64
        // tiles (512 workgroups at N = 32768) beat 128x128 by 17%; a long-K
        // product with both operands k-contiguous runs best on 64x64 tiles
        // split to about 256 workgroups (30%); an M-major weight with many
        // output columns on unsplit 64x128 tiles (25%); otherwise the deep
        // 128x128 ring, split along K to fill the CUs.
        const long rows64 = (d.M + 63) / 64;
        if (d.beta && d.b_kmajor && (long)((d.N + 63) / 64) * ((d.M + 127) / 128) >= 256 && tile_fits(d, 20))
            return Choice{20, 1};
        if (d.a_kmajor && d.b_kmajor && tile_fits(d, 19)) {
            const long tiles = rows64 * ((d.N + 63) / 64);
            int sp = 1;
            while (sp < 64 && tiles * sp < 256 && d.K / (2 * sp) >= 256) sp *= 2;
            if (sp == 1 || !d.beta) return Choice{19, sp};
        }
        if (d.a_kmajor && !d.b_kmajor && rows64 * (d.N / 128) >= 128 && tile_fits(d, 18)) return Choice{18, 1};
        return Choice{16, model_splits(d, 128, 128, 1, 64)};
    }
    if (es == 2 && d.a_kmajor && d.M > 256 && d.M <= 1024 && tile_fits(d, 18)) {
        // few rows (the time-parallel products at 16 batch rows: 800): 64x128
        // tiles at two workgroups per CU fill more of the chip than 128-row
        // tiles; measured at 800 x 4096 x 1024 (input projection) 23.7 -> 18.4
        // us and 800 x 1024 x 4096 (dX) 27.5 -> 22.7 us; from 1600 rows on the
        // 128-row tiles are faster.  Split along K to fill the CUs (dX: 4).
        return Choice{18, model_splits(d, 64, 128, kTileSlots[18], kTileKD[18])};
    }
    const double cu_rate = 4096.0 * 2.4e9 * 0.7;   // FLOP/s of one CU at a realistic fraction
    if (es == 2 && d.a_kmajor && d.K >= 16384 && tile_fits(d, 22)) {
        // a very long K over few output tiles (BigLSTM's dX, K = 4H = 32768):
        // 256x256 tiles split along K to about one workgroup per CU.  Measured
        // at 2560 x 1024 x 32768: 243 us with 128x128 tiles as the model splits
        // them, 193 us on 256x128 split 3 ways, 170 us on 256x256 split 6 ways
        const long tiles = (long)((d.M + 255) / 256) * ((d.N + 255) / 256);
        if (tiles <= 128) {
            int sp = (int)(256 / tiles);
            if (sp > 8) sp = 8;
            while (sp > 1 && d.K / sp < 2048) --sp;
            return Choice{22, sp};
        }
    }
    if (es == 2 && d.a_kmajor && !d.b_kmajor && tile_fits(d, 22)) {
        // dX = dZ W: 256x256 tiles of 16 waves once they occupy three quarters
        // of the CUs.  Measured: GNMT-4 B = 256 (200 tiles) 142 -> 107 us,
        // B = 512 269 -> 216 us, GNMT-8 155 -> 119 us; at B = 128 (100 tiles)
        // they lose (65.6 -> 71.2 us)
        const long tiles = (long)((d.M + 255) / 256) * ((d.N + 255) / 256);
        if (tiles >= 192) return Choice{22, 1};
    }
    if (es == 2 && d.a_kmajor && d.b_kmajor && tile_fits(d, 22)) {
        // both operands k-contiguous (the input projection) with enough
        // 256x256 tiles to occupy most CUs: one 16-wave workgroup per CU
        // loads a third fewer operand bytes from L2 per product than two
        // 128x256 workgroups, the limit of those.  Measured: 6400 x 4096 x
        // 1024 89 -> 74 us, 3200 rows 44 -> 38 us, 25600 rows 387 -> 321 us,
        // K = 2048 339 -> 287 us, 2560 x 32768 x 1024 285 -> 237 us; with
        // 1600 rows (112 tiles) 29.5 -> 34.6 us, so not below ~192 tiles.
        const long tiles = (long)((d.M + 255) / 256) * ((d.N + 255) / 256);
        if (tiles >= 192) return Choice{22, 1};
    }
    if (es == 2 && d.a_kmajor && d.b_kmajor && dl_ok(d, 128, 256, 1)) {
        // both operands k-contiguous (the input projection): 128x256 tiles of
        // 8 waves move less L2 traffic per flop than 128x128 once they fill
        // the 512 workgroup slots at least once
        const long tiles = (long)((d.M + 127) / 128) * ((d.N + 255) / 256);
        if (tiles >= 512) return Choice{2, 1};
    }
    if (es == 2 && dl_ok(d, 128, 128, 1)) {
        // direct-to-LDS 128x128 tiles run two workgroups per CU (512 slots);
        // split K only to fill the slots.  dX's layout takes 64-deep stages in
        // a ring of two (B = 128 65.6 -> 64.1 us, B = 64 44.8 -> 42.7 us), the
        // other products 32-deep stages in a ring of four
        const int t128 = (d.a_kmajor && !d.b_kmajor && tile_fits(d, 5)) ? 5 : 3;
        Choice best{t128, 1};
        double best_t = 1e30;
        const long tiles = (long)((d.M + 127) / 128) * ((d.N + 127) / 128);
        for (int sp = 1; sp <= 64; sp *= 2) {   // skinny products (per-step recurrences) split K widely
            if (sp > 1 && (!d.splitk_ws || (size_t)sp * d.M * d.N > d.splitk_ws_floats)) break;
            if (sp > 1 && d.K / sp < 256) break;
            const long items = tiles * sp;
            const long waves = (items + 511) / 512;
            double tt = waves * 2.0 * 128 * 128 * ((double)d.K / sp) / (cu_rate * 0.5);
            if (sp > 1) tt += ((double)sp + 1.0) * d.M * d.N * 4.0 / 5.0e12;
            if (tt < best_t * 0.97) {
                best_t = tt;
                best = Choice{t128, sp};
            }
        }
        return best;
    }
    const int cus = 256;
    Choice best{3, 1};
    double best_t = 1e30;
    for (int t = 0; t < 4; ++t) {
        if (es == 4 && t != 3) continue;            // fp32 inputs: the 128x128 tile only
        const long tiles = (long)((d.M + BMs[t] - 1) / BMs[t]) * ((d.N + BNs[t] - 1) / BNs[t]);
        for (int sp = 1; sp <= 8; sp *= 2) {
            if (sp > 1 && (!d.splitk_ws || (size_t)sp * d.M * d.N > d.splitk_ws_floats)) break;
            if (sp > 1 && d.K / sp < 512) break;
            const long items = tiles * sp;
            const long waves = (items + cus - 1) / cus;
            const double item_t = 2.0 * BMs[t] * BNs[t] * ((double)d.K / sp) / (cu_rate * eff[t]);
            double tt = waves * item_t;
            if (sp > 1) tt += ((double)sp + 1.0) * d.M * d.N * 4.0 / 5.0e12;
            if (tt < best_t * 0.97) {
                best_t = tt;
                best = Choice{t, sp};
            }
        }
    }
    return best;
}

// The direct-to-LDS kernel needs whole 32-deep K stages and, for an operand
// whose rows are the contiguous dimension in memory, whole tiles of rows.
bool dl_ok(const GemmDesc &d, int BM, int BN, int splits)
{
    const char *env = std::getenv("LSTM355_GEMM_DL");
    if (env && env[0] == '0') return false;
    if (d.K % 32 && (d.a_kmajor || d.b_kmajor)) return false;   // a partial last stage needs k as the row index
    if (!d.a_kmajor && d.M % BM) return false;
    if (!d.b_kmajor && d.N % BN) return false;
    const long ea = d.a_kmajor ? (long)d.M * d.lda : (long)d.K * d.lda;
    const long eb = d.b_kmajor ? (long)d.N * d.ldb : (long)d.K * d.ldb;
    if (ea * 2 > 0x7fffffffL || eb * 2 > 0x7fffffffL) return false;
    (void)splits;
    return true;
}

// Largest split count <= want whose fp32 partials fit the caller's split-K workspace.
int fit_splits(const GemmDesc &d, int want)
{
    int sp = want < 1 ? 1 : want;   // 0 (no request) means one
    while (sp > 1 && (!d.splitk_ws || (size_t)sp * (size_t)d.M * (size_t)d.N > d.splitk_ws_floats)) --sp;
    return sp;
}

template <typename TO, bool AK, bool BKM>
hipError_t launch_tile(int tile, const GemmDesc &d, int splits, hipStream_t s)
{
    if (d.beta && splits <= 1) {   // accumulating into C: the 128x128 configurations with staged C reads
        if (tile == 16 && d.K % 64 == 0) return launch_gemm_dl<TO, 128, 128, AK, BKM, 64, 4, 2, 2, true>(d, 1, s);
        if (tile == 5 && d.K % 64 == 0) return launch_gemm_dl<TO, 128, 128, AK, BKM, 64, 2, 2, 2, true>(d, 1, s);
        if (tile == 3 || tile == 5 || tile == 16) return launch_gemm_dl<TO, 128, 128, AK, BKM, 32, 4, 2, 2, true>(d, 1, s);
        if constexpr (AK && BKM) {
            if (tile == 19 && d.K % 64 == 0) return launch_gemm_dl<TO, 64, 64, AK, BKM, 64, 4, 2, 2, true>(d, 1, s);
            if (tile == 20 && d.K % 64 == 0) return launch_gemm_dl<TO, 128, 64, AK, BKM, 64, 3, 2, 2, true>(d, 1, s);
        }
    }
    switch (tile) {
    case 0: return launch_gemm_dl<TO, 256, 256, AK, BKM, 32, 4, 2, 4>(d, splits, s);
    case 1: return launch_gemm_dl<TO, 256, 128, AK, BKM, 32, 3, 4, 2>(d, splits, s);
    case 2: return launch_gemm_dl<TO, 128, 256, AK, BKM, 32, 3, 2, 4>(d, splits, s);
    case 4: return launch_gemm_dl<TO, 256, 256, AK, BKM, 32, 4, 4, 2>(d, splits, s);
    case 5: return launch_gemm_dl<TO, 128, 128, AK, BKM, 64, 2, 2, 2>(d, splits, s);
    case 6: return launch_gemm_dl<TO, 256, 128, AK, BKM, 64, 2, 4, 2>(d, splits, s);
    case 7: return launch_gemm_dl<TO, 128, 256, AK, BKM, 64, 2, 2, 4>(d, splits, s);
    case 8: return launch_gemm_dl<TO, 256, 256, AK, BKM, 64, 2, 2, 4>(d, splits, s);
    case 9: return launch_gemm_dl<TO, 256, 256, AK, BKM, 32, 4, 2, 2>(d, splits, s);
    case 10: return launch_gemm_dl<TO, 256, 256, AK, BKM, 64, 2, 2, 2>(d, splits, s);
    case 11: return launch_gemm_dl<TO, 128, 256, AK, BKM, 32, 3, 2, 2>(d, splits, s);
    case 12: return launch_gemm_dl<TO, 256, 128, AK, BKM, 32, 3, 2, 2>(d, splits, s);
    case 13: return launch_gemm_dl<TO, 128, 256, AK, BKM, 64, 3, 2, 4>(d, splits, s);
    case 14: return launch_gemm_dl<TO, 256, 128, AK, BKM, 64, 3, 4, 2>(d, splits, s);
    case 15: return launch_gemm_dl<TO, 128, 128, AK, BKM, 64, 3, 2, 2>(d, splits, s);
    case 16: return launch_gemm_dl<TO, 128, 128, AK, BKM, 64, 4, 2, 2>(d, splits, s);
    case 17: return launch_gemm_dl<TO, 128, 128, AK, BKM, 32, 8, 2, 2>(d, splits, s);
    case 18:
        if constexpr (AK) return launch_gemm_dl<TO, 64, 128, AK, BKM, 64, 3, 2, 2>(d, splits, s);
        return hipErrorInvalidValue;
    case 19:
        if constexpr (AK && BKM) return launch_gemm_dl<TO, 64, 64, AK, BKM, 64, 4, 2, 2>(d, splits, s);
        return hipErrorInvalidValue;
    case 20:
        if constexpr (BKM) return launch_gemm_dl<TO, 128, 64, AK, BKM, 64, 3, 2, 2>(d, splits, s);
        return hipErrorInvalidValue;
    case 21: return launch_gemm_dl<TO, 256, 256, AK, BKM, 32, 4, 4, 4>(d, splits, s);
    case 22: return launch_gemm_dl<TO, 256, 256, AK, BKM, 64, 2, 4, 4>(d, splits, s);
    case 23: return launch_gemm_dl<TO, 256, 128, AK, BKM, 64, 3, 4, 4>(d, splits, s);
    case 24: return launch_gemm_dl<TO, 128, 256, AK, BKM, 64, 3, 4, 4>(d, splits, s);
    default: return launch_gemm_dl<TO, 128, 128, AK, BKM, 32, 4, 2, 2>(d, splits, s);
    }
}

// Whether tile configuration `t` can run descriptor `d` (whole k stages,
// whole tiles along an operand whose rows are contiguous in memory, whole
// tiles per column block).
bool tile_fits(const GemmDesc &d, int t)
{
    if (t < 0 || t >= NTILES) return false;
    const int kd = kTileKD[t];
    if (d.K % kd && (d.a_kmajor || d.b_kmajor)) return false;
    if ((!d.a_kmajor && kTileBM[t] < 128) || (!d.b_kmajor && kTileBN[t] < 128)) return false;
    if (d.N1 > 0 && (d.N1 % kTileBN[t] || d.N % kTileBN[t] || d.M % kTileBM[t])) return false;
    if (d.N1 > 0 && d.B3 && (d.ylo % kd || d.yhi % kd || d.hlo % kd || d.hlen % kd))
        return false;   // stages stay in one segment
    return dl_ok(d, kTileBM[t], kTileBN[t], 1);
}

// Tuning override from the environment: "tile" or "tile,splits", in
// LSTM355_GEMM_TILE_<class number> for one kernel class, else
// LSTM355_GEMM_TILE for every product.
thread_local int g_kclass = -1;

bool env_choice(Choice *c)
{
    char name[40];
    std::snprintf(name, sizeof(name), "LSTM355_GEMM_TILE_%d", g_kclass);
    const char *env = std::getenv(name);
    if (!env) env = std::getenv("LSTM355_GEMM_TILE");
    if (!env) return false;
    int t = std::atoi(env), sp = 0;
    const char *comma = std::strchr(env, ',');
    if (comma) sp = std::atoi(comma + 1);
    if (t < 0 || t >= NTILES || sp < 0) return false;
    *c = Choice{t, sp};
    return true;
}

template <typename TI, typename TO, bool AK, bool BKM>
hipError_t dispatch_tiles(const GemmDesc &d, hipStream_t s)
{
    if constexpr (sizeof(TI) == 2 && !AK && !BKM) {
        if (d.N1 > 0) {   // two column blocks: no split; 128x128 tiles, 64-deep stages where they fit
            Choice c{5, 1};
            // 256x256 tiles of 16 waves once the launch's tiles fill the CUs at
            // least once (BigLSTM's 32768 x 2048 product: 368 -> 324 us; the
            // layer wavefront's four 4096 x 2048 products in one launch: 73.7 ->
            // 69.8 us at B = 16, 123.9 -> 109.7 us at B = 32; one 4096-row
            // product's 128 tiles leave half the CUs idle)
            const long nb = d.nbatch > 1 ? d.nbatch : 1;
            if ((long)(d.M / 256) * (d.N / 256) * nb >= 256 && tile_fits(d, 22)) c.tile = 22;
            env_choice(&c);
            if (!tile_fits(d, c.tile)) c.tile = 5;
            if (!tile_fits(d, c.tile)) c.tile = 3;
            if (!tile_fits(d, c.tile)) return hipErrorInvalidValue;
            return launch_tile<TO, AK, BKM>(c.tile, d, 1, s);
        }
    }
    if (d.N1 > 0) return hipErrorInvalidValue;
    Choice c = choose(d, sizeof(TI));
    if (d.partials > 1) {   // exactly the requested parts, all of them in the workspace
        if (d.nbatch > 1 || fit_splits(d, d.partials) != d.partials) return hipErrorInvalidValue;
        c.splits = d.partials;
    }
    c.splits = fit_splits(d, c.splits);   // also bounds a tuning override
    if constexpr (sizeof(TI) == 4) {
        return launch_gemm<TI, TO, 128, 128, 64, AK, BKM>(d, c.splits, s);
    } else {
        if (tile_fits(d, c.tile)) return launch_tile<TO, AK, BKM>(c.tile, d, c.splits, s);
        if (dl_ok(d, 128, 128, c.splits)) return launch_tile<TO, AK, BKM>(3, d, c.splits, s);
        switch (c.tile) {
        case 0: return launch_gemm<TI, TO, 256, 256, 128, AK, BKM>(d, c.splits, s);
        case 1: return launch_gemm<TI, TO, 256, 128, 128, AK, BKM>(d, c.splits, s);
        case 2: return launch_gemm<TI, TO, 128, 256, 128, AK, BKM>(d, c.splits, s);
        default: return launch_gemm<TI, TO, 128, 128, 128, AK, BKM>(d, c.splits, s);
        }
    }
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

bool gemm_dual_ok(const GemmDesc &d)
{
    if (d.in != DType::BF16 || d.a_kmajor || d.b_kmajor || !d.out_f32) return false;
    if (d.N1 <= 0 || d.N1 >= d.N || d.N1 % 128 || d.N % 128 || d.M % 128) return false;
    if (d.ylo < 0 || d.yhi > d.K || d.ylo >= d.yhi) return false;
    // with an h0 segment, stages of 32 k must not straddle a segment boundary;
    // without one, the second block runs over [ylo, yhi) alone
    if (d.B3 && (d.K % 32 || d.ylo % 32 || d.yhi % 32 || d.hlo % 32 || d.hlen % 32)) return false;
    if (d.B3 && (d.hlo < 0 || d.hlo + d.hlen > d.K)) return false;
    return dl_ok(d, 128, 128, 1);
}

// fp16 C only where the product takes the 256x256 tile unsplit (the same
// shapes on which choose() picks it: more than 1024 rows, at least 192 tiles).
bool gemm_f16_ok(const GemmDesc &d)
{
    if (d.in != DType::BF16 || !d.a_kmajor || !d.b_kmajor || d.out_f32 || d.beta || d.N1 > 0 || d.cell_h > 0 ||
        d.nbatch > 1 || d.partials > 0 || d.M <= 1024)
        return false;
    const long tiles = (long)((d.M + 255) / 256) * ((d.N + 255) / 256);
    return tiles >= 192 && tile_fits(d, 22);
}

bool gemm_cell_ok(const GemmDesc &d)
{
    if (d.cell_h <= 0 || d.in != DType::BF16 || !d.a_kmajor || !d.b_kmajor || !d.out_f32 || !d.beta) return false;
    if (d.N1 > 0 || d.bias || !d.cell_c || !d.cell_m || d.N != 4 * d.cell_h || d.cell_h % 16 || d.K % 64) return false;
    return dl_ok(d, 128, 64, 1);
}

hipError_t gemm(const GemmDesc &d, hipStream_t s, int kclass)
{
    if (d.M <= 0 || d.N <= 0 || d.K <= 0) return hipSuccess;
    if (d.partials > 1 && (d.N1 > 0 || d.cell_h > 0 || d.nbatch > 1 || !d.splitk_ws)) return hipErrorInvalidValue;
    const double es = (double)dsize(d.in);
    double flops, bytes;
    if (d.N1 > 0) {   // second column block over its own k range
        const double k2 = (double)(d.yhi - d.ylo) + (d.B3 ? d.hlen : 0);
        flops = 2.0 * d.M * ((double)d.N1 * d.K + (double)(d.N - d.N1) * k2);
        bytes = es * ((double)d.M * d.K + (double)d.N1 * d.K + (double)(d.N - d.N1) * k2) +
                4.0 * d.M * d.N * (d.beta ? 2.0 : 1.0);
    } else {
        flops = 2.0 * d.M * d.N * (double)d.K;
        bytes = es * ((double)d.M * d.K + (double)d.N * d.K) +
                (d.out_f32 ? 4.0 : es) * (double)d.M * d.N * (d.beta ? 2.0 : 1.0);
    }
    if (d.cell_h > 0) {   // the cell update's own traffic: read cprev, write activations, c, m
        if (!gemm_cell_ok(d)) return hipErrorInvalidValue;
        bytes += (double)d.M * d.cell_h * (4.0 * (d.cell_prev ? 1 : 0) + 4.0 + 2.0 + (d.cell_cT ? 4.0 : 0.0));
    }
    if (d.nbatch > 1) {
        flops *= d.nbatch;
        bytes *= d.nbatch;
    }
    ProfScope ps(kclass, s, flops, bytes);
    g_kclass = kclass;
    if (d.cell_h > 0) return launch_gemm_dl<float, 128, 64, true, true, 64, 3, 2, 2, true, true>(d, 1, s);
    if (d.out_f16) {
        if (!gemm_f16_ok(d)) return hipErrorInvalidValue;
        return launch_gemm_dl<f16_t, 256, 256, true, true, 64, 2, 4, 4>(d, 1, s);
    }
    return d.in == DType::BF16 ? dispatch_layout<bf16_t>(d, s) : dispatch_layout<float>(d, s);
}

}  // namespace lstm355
