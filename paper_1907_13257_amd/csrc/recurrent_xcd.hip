// recurrent_xcd.hip -- persistent forward / BPTT recurrences whose per-step
// exchange stays inside one XCD (bf16, plain LSTM, H in {256, 512, 1024}).
//
// The MI355X has 8 XCDs of 32 CUs, each XCD with its own L2; a 256-workgroup
// launch puts 32 workgroups on each XCD, and a workgroup takes the XCD it
// finds itself on (XCC_ID register) as its own.  XCD x owns batch rows [x*RX, x*RX + RX), RX = ceil(B/8),
// and all H cells of those rows: its 32 workgroups each own HN = H/32 cells.
// The rows of h_{t-1} (forward) and of dz_t (backward) that a workgroup needs
// are therefore produced inside its own XCD and travel through that XCD's
// L2 only.  Every workgroup keeps its share of the recurrent weights in
// registers for the whole kernel: forward, the 4*HN rows of R feeding its
// cells (256 KiB at H = 1024, 32 KiB per wave); backward, the HN columns of R
// (rows of R^T).
//
// Exchange protocol per step (no barrier between workgroups, no flags, no
// cache flushes): the exchanged rows (y, or dz) are filled with a NOT_READY
// pattern before the launch, and every element is written exactly once with
// a plain store.  A consumer wave copies its slice of the rows it needs from
// L2 into LDS with loads that miss its CU's L1, and repeats the copy until no
// element of its valid rows still holds NOT_READY.  Nothing is waited on by
// producers, and a consumer proceeds as soon as the values it uses are
// there.  Every wait has a wall-clock watchdog and an abort word, so every
// wave exits.
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"

namespace lstm355 {

// Sticky error bits of this translation unit's kernels (TRIP_* values).
__device__ unsigned g_xcd_tripped = 0;

namespace {

constexpr int XT = 512;          // threads per workgroup (8 waves, 2 per SIMD)
constexpr int NXCD = 8;
constexpr int WG_PER_XCD = 32;
constexpr int HWREG_XCC_ID = (31 << 11) | (0 << 6) | 20;   // s_getreg: XCC_ID, 32 bits

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *p)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, 0x7fffffff, 0x00020000);
}

// Role of a workgroup: its XCD is the one it runs on (XCC_ID register) and
// its slot within the XCD is blockIdx.x / 8.  Dispatch hands workgroups to
// the XCDs in turn, so the XCD of workgroup w is (w + o) % 8 for an offset o
// that depends on earlier dispatches; the 32 workgroups of an XCD then have
// distinct slots.  Each workgroup claims its slot in a per-XCD bit mask; a
// slot claimed twice means the roles do not cover every (XCD, slot) pair, and
// the launch is abandoned (abort word set, placement error recorded).
__device__ __forceinline__ bool claim_role(unsigned *flags, int *s_xcd)
{
    if (threadIdx.x == 0) {
        const int x = (int)(__builtin_amdgcn_s_getreg(HWREG_XCC_ID) & 7u);
        const unsigned bit = 1u << (blockIdx.x >> 3);
        const unsigned prev =
            __hip_atomic_fetch_or(flags + XCD_CLAIM + x, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (prev & bit) {
            __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_PLACEMENT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(flags + XCD_ABORT, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            *s_xcd = -1;
        } else {
            *s_xcd = x;
        }
    }
    __syncthreads();
    return *s_xcd >= 0;
}

// Staging of exchanged rows.  Each wave copies the rows it multiplies (16
// batch rows, its own k range of RB bytes per row) from the XCD's L2 into its
// own LDS tile with buffer->LDS loads of whole 128-byte lines, then reads MFMA
// fragments from the tile.  16-byte chunk c of row r sits at slot
// c ^ swz(r), which puts the 16 rows one fragment read touches in distinct
// LDS banks (a 256-byte window of 64 four-byte banks).
template <int RB>
__device__ __forceinline__ int stage_swz(int r)
{
    if constexpr (RB >= 256)
        return r & 15;
    else
        return (r / (256 / RB)) % (RB / 16);
}

// Copies rows [r0, r0+16) x bytes [kbyte, kbyte+RB) of a row-major bf16 matrix
// (row pitch ld elements, descriptor `rs`) into the wave's tile at LDS byte
// `tile` (16*RB bytes).  Rows past the descriptor's end read as zero.  ROT:
// the 1 KiB instructions are issued starting at `rot` (mod their count), so
// that the workgroups of an XCD, which all copy the same rows, start on
// different lines of L2 (measured: 2% faster for the forward's four
// instructions per wave, slower for the backward's sixteen).
template <int RB, bool COHERENT = false, bool ROT = false>
__device__ __forceinline__ void stage_rows(u32x4 rs, long r0, long ld, int kbyte, unsigned tile, int lane,
                                           unsigned qmask = ~0u, int rot = 0)
{
    static_assert(RB % 64 == 0 && (16 * RB) % 1024 == 0, "whole 1 KiB instructions");
    constexpr int NQ = 16 * RB / 1024;
    static_assert((NQ & (NQ - 1)) == 0, "a power of two of instructions");
#pragma unroll
    for (int qi = 0; qi < NQ; ++qi) {
        const int q = ROT ? (qi + rot) & (NQ - 1) : qi;
        if (!((qmask >> q) & 1u)) continue;   // wave-uniform
        const int o = q * 1024 + lane * 16;
        const int r = o / RB, p = (o % RB) >> 4;
        const int c = p ^ stage_swz<RB>(r);
        const unsigned voff = (unsigned)((r0 + r) * ld * 2 + kbyte + c * 16);
        if (COHERENT)
            dma16_sc1(rs, __builtin_amdgcn_readfirstlane(tile + q * 1024), voff);
        else
            dma16(rs, __builtin_amdgcn_readfirstlane(tile + q * 1024), voff);
    }
}

// Fragment of 32-deep k chunk `cc` for MFMA operand row lane%16.
template <int RB>
__device__ __forceinline__ u32x4 stage_frag(const char *tile, int cc, int lane)
{
    const int i = lane & 15;
    const int slot = (cc * 4 + (lane >> 4)) ^ stage_swz<RB>(i);
    return *reinterpret_cast<const u32x4 *>(tile + i * RB + slot * 16);
}

__device__ __forceinline__ void wait_own_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void wait_own_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Exchanged bf16 rows are filled with NOT_READY before the launch and each
// element is written exactly once, never with that pattern (a NaN of that
// encoding is replaced by the canonical quiet NaN).  A consumer therefore
// knows an element is final once it reads anything else.
constexpr bf16_t NOT_READY = XCD_NOT_READY;

__device__ __forceinline__ bf16_t ready_value(bf16_t v) { return v == NOT_READY ? (bf16_t)0x7fc0u : v; }

// Running per-half maximum of the bf16 patterns a lane has read: NOT_READY
// (0xffff) is the largest 16-bit value, so a lane read one exactly when a
// half of its maximum is 0xffff.  Four packed max operations per fragment.
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u16x2 max_halves(u16x2 m, u32x4 v)
{
    const u16x2 a = __builtin_elementwise_max(__builtin_bit_cast(u16x2, v[0]), __builtin_bit_cast(u16x2, v[1]));
    const u16x2 b = __builtin_elementwise_max(__builtin_bit_cast(u16x2, v[2]), __builtin_bit_cast(u16x2, v[3]));
    return __builtin_elementwise_max(m, __builtin_elementwise_max(a, b));
}

__device__ __forceinline__ bool saw_not_ready(u16x2 m) { return m.x == NOT_READY || m.y == NOT_READY; }

// acc[i] = (16 exchanged rows, this wave's k range) x rf[i] on the matrix
// cores (WT: the transposed product, rf[i] x the rows), once every element of
// the first `valid` rows is final.  Each attempt
// copies the wave's slice from the XCD's L2 into its LDS tile (L1 bypassed)
// and multiplies it while checking for NOT_READY; an attempt that saw one is
// discarded and repeated.  Returns false if another workgroup aborted or the
// wall-clock watchdog expired (then the abort word is raised).
template <int RB, int KCW, int NBX, bool WT = false>
__device__ __forceinline__ bool stage_mma_when_ready(u32x4 rs, long r0, long ld, int kbyte, unsigned tile,
                                                     const char *tilep, int lane, int valid,
                                                     const u32x4 (&rf)[NBX][KCW], f32x4 (&acc)[NBX],
                                                     unsigned *flags, unsigned long long timeout, int rot)
{
    constexpr int RPI = 1024 / RB > 0 ? 1024 / RB : 1;   // rows per 1 KiB instruction (RB <= 1024)
    static_assert(RB <= 1024, "one row per instruction at most");
    const __amdgpu_buffer_rsrc_t rfl = rsrc(flags);
    const bool row_in = (lane & 15) < valid;
    const unsigned long long t0 = wall_clock64();
    // copy only the instructions that cover valid rows (an XCD may own fewer
    // than 16 rows); the other rows of the tile feed only discarded outputs
    unsigned qmask = 0;
#pragma unroll
    for (int q = 0; q < 16 / RPI; ++q)
        if (q * RPI < valid) qmask |= 1u << q;
    while (true) {
        stage_rows<RB, true, WT>(rs, r0, ld, kbyte, tile, lane, qmask, rot);
        const unsigned ab = __builtin_amdgcn_raw_buffer_load_b32(rfl, XCD_ABORT * 4, 0, 16);
        wait_own_loads();
#pragma unroll
        for (int i = 0; i < NBX; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        u16x2 seen = {0, 0};
#pragma unroll
        for (int c = 0; c < KCW; ++c) {
            // fragments in flight at most four chunks ahead (bounded registers)
            if (c % 4 == 0 && c > 0) __builtin_amdgcn_sched_barrier(0);
            const u32x4 fa = stage_frag<RB>(tilep, c, lane);
            seen = max_halves(seen, fa);
#pragma unroll
            for (int i = 0; i < NBX; ++i) {
                if (WT)
                    mfma16(acc[i], rf[i][c], fa, bf16_t{});
                else
                    mfma16(acc[i], fa, rf[i][c], bf16_t{});
            }
        }
        const unsigned long long lm = __builtin_amdgcn_ballot_w64(saw_not_ready(seen) && row_in);
        if (lm == 0) return true;
        // re-copy only the instructions that cover rows still incomplete
        const unsigned rows = (unsigned)(lm | (lm >> 16) | (lm >> 32) | (lm >> 48)) & 0xffffu;
        qmask = 0;
#pragma unroll
        for (int q = 0; q < 16 / RPI; ++q)
            if ((rows >> (q * RPI)) & ((1u << RPI) - 1u)) qmask |= 1u << q;
        if (ab != 0) return false;
        if (wall_clock64() - t0 > timeout) {
            if (lane == 0) {
                __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_WATCHDOG, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(flags + XCD_ABORT, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            return false;
        }
        wait_own_lds();
    }
}

// Chunked staging: a wave's slice (16 rows x KCW 32-deep k chunks) is copied
// in pairs of chunks, 64 k values = 128 bytes per row: pair p goes to LDS
// block p (2 KiB, row i at byte 128*i), with two 1 KiB instructions of 8
// whole rows each, so a wave can multiply the first pairs while the later
// ones are still on their way.  Lane l of instruction h moves 16-byte piece
// l % 8 of row 8h + l/8; within a row, piece P sits at slot P ^ ((row/2) % 8),
// which puts the 16 rows that one fragment read touches in distinct banks.
// Rows at or past `valid` are not copied (an offset past the descriptor's end
// loads zeros).
constexpr unsigned OOB_OFFSET = 0x80000000u;

__device__ __forceinline__ unsigned pair_voff(long r0, long ld, int kbyte, int lane, int h, int valid)
{
    const int r = 8 * h + (lane >> 3), piece = (lane & 7) ^ ((r >> 1) & 7);
    return r < valid ? (unsigned)((r0 + r) * ld * 2 + kbyte + piece * 16) : OOB_OFFSET;
}

__device__ __forceinline__ u32x4 pair_frag(const char *tilep, int c, int lane)
{
    const int i = lane & 15, piece = 4 * (c & 1) + (lane >> 4);
    return *reinterpret_cast<const u32x4 *>(tilep + (c >> 1) * 2048 + i * 128 + ((piece ^ ((i >> 1) & 7)) * 16));
}

// s_waitcnt vmcnt(n), n in [0, 15]; n is a constant once the caller's loop
// is unrolled, and the switch folds to the one instruction.
__device__ __forceinline__ void wait_loads_upto(int n)
{
#define LSTM355_VMCNT(N)                                      \
    case N:                                                   \
        asm volatile("s_waitcnt vmcnt(" #N ")" ::: "memory"); \
        break;
    switch (n) {
        LSTM355_VMCNT(0) LSTM355_VMCNT(1) LSTM355_VMCNT(2) LSTM355_VMCNT(3)
        LSTM355_VMCNT(4) LSTM355_VMCNT(5) LSTM355_VMCNT(6) LSTM355_VMCNT(7)
        LSTM355_VMCNT(8) LSTM355_VMCNT(9) LSTM355_VMCNT(10) LSTM355_VMCNT(11)
        LSTM355_VMCNT(12) LSTM355_VMCNT(13) LSTM355_VMCNT(14)
        default: asm volatile("s_waitcnt vmcnt(15)" ::: "memory"); break;
    }
#undef LSTM355_VMCNT
}

// The pipelined form of stage_mma_when_ready (untransposed product): all
// copies are issued at once (two instructions per chunk pair, KCW in all);
// each group of G chunks is multiplied as soon as its own copies have landed
// and none of its valid elements holds NOT_READY.  A group that saw one is copied again together
// with every later pair (they were copied at the same time, so they are
// likely stale too), until it is complete.  Chunks are multiplied in order,
// so the sums are those of the unpipelined form, bit for bit.
template <int KCW, int NBX, int G>
__device__ __forceinline__ bool stage_mma_pipe(u32x4 rs, long r0, long ld, int kbyte, unsigned tile,
                                               const char *tilep, int lane, int valid,
                                               const u32x4 (&rf)[NBX][KCW], f32x4 (&acc)[NBX], unsigned *flags,
                                               unsigned long long timeout)
{
    static_assert(KCW >= 2 && KCW <= 16 && KCW % 2 == 0, "whole chunk pairs, at most 16 instructions in flight");
    static_assert(G % 2 == 0 && KCW % G == 0, "whole pairs per group, whole groups");
    const unsigned v0 = pair_voff(r0, ld, kbyte, lane, 0, valid);
    const unsigned v1 = pair_voff(r0, ld, kbyte, lane, 1, valid);
    const bool row_in = (lane & 15) < valid;
    auto issue_from = [&](int p0) {
#pragma unroll
        for (int p = 0; p < KCW / 2; ++p) {
            if (p < p0) continue;
            const unsigned blk = tile + p * 2048;
            dma16_sc1(rs, __builtin_amdgcn_readfirstlane(blk), v0 + p * 128);
            dma16_sc1(rs, __builtin_amdgcn_readfirstlane(blk + 1024), v1 + p * 128);
        }
    };
    issue_from(0);
#pragma unroll
    for (int i = 0; i < NBX; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const __amdgpu_buffer_rsrc_t rfl = rsrc(flags);
    unsigned long long t0 = 0;
    bool waited = false;
#pragma unroll
    for (int c0 = 0; c0 < KCW; c0 += G) {
        // the newest instructions are always the copies of pairs c0/2 .. KCW/2-1
        wait_loads_upto(KCW - G - c0);
        u32x4 fa[G];
        u16x2 seen = {0, 0};
#pragma unroll
        for (int g = 0; g < G; ++g) {
            fa[g] = pair_frag(tilep, c0 + g, lane);
            seen = max_halves(seen, fa[g]);
        }
        while (__builtin_amdgcn_ballot_w64(saw_not_ready(seen) && row_in) != 0) {
            if (!waited) {
                t0 = wall_clock64();
                waited = true;
            }
            const unsigned ab = __builtin_amdgcn_raw_buffer_load_b32(rfl, XCD_ABORT * 4, 0, 16);
            wait_own_loads();
            if (ab != 0) return false;
            if (wall_clock64() - t0 > timeout) {
                if (lane == 0) {
                    __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_WATCHDOG, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(flags + XCD_ABORT, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                return false;
            }
            wait_own_lds();   // the fragments are in registers before their blocks are overwritten
            issue_from(c0 / 2);
            wait_loads_upto(KCW - G - c0);
            seen = u16x2{0, 0};
#pragma unroll
            for (int g = 0; g < G; ++g) {
                fa[g] = pair_frag(tilep, c0 + g, lane);
                seen = max_halves(seen, fa[g]);
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int i = 0; i < NBX; ++i) mfma16(acc[i], fa[g], rf[i][c0 + g], bf16_t{});
    }
    return true;
}

// The dz rows of a BPTT step times the resident R^T rows, for the per-layer
// backward.  With two or more row blocks per XCD the copy is pipelined in two
// halves (GNMT-4, B = 256: 336 -> 307 us per layer); with one, the first copy
// usually finds rows still missing, and re-copying just the missing rows
// after one full copy is faster (163 -> 170 us when pipelined).  The layer
// wavefront's two row blocks (17 to 32 rows in one XCD) lose with it too
// (B = 32: 355 -> 367 us), and keep the unpipelined copy.
template <int RB, int KCW, int NBB, int MBX>
__device__ __forceinline__ bool stage_dz(u32x4 rs, long r0, long ld, int kbyte, unsigned tile, const char *tilep,
                                         int lane, int valid, const u32x4 (&rf)[NBB][KCW], f32x4 (&acc)[NBB],
                                         unsigned *flags, unsigned long long timeout, int rot)
{
    if constexpr (MBX >= 2)
        return stage_mma_pipe<KCW, NBB, KCW / 2>(rs, r0, ld, kbyte, tile, tilep, lane, valid, rf, acc, flags,
                                                        timeout);
    else
        return stage_mma_when_ready<RB, KCW, NBB>(rs, r0, ld, kbyte, tile, tilep, lane, valid, rf, acc, flags,
                                                  timeout, rot);
}

// Resident columns of a row-major bf16 matrix M [rows][ld] (R or W, whose
// columns are the rows of R^T or W^T that the backward kernels multiply by):
// for lane L, rf[i][c] = M[k0 + 32c + 8(L/16) + e][j0 + 16i + L%16], e = 0..7,
// zero for a column at or past HN.  The wave copies its KW x NC block of M
// into its LDS tile (NBB passes of KW/NBB k-rows, 2*NC bytes per k-row) and
// reads the fragments with ds_read_b64_tr_b16: in each group of 16 lanes,
// source lane s addresses 8 bytes at (k-row kb + s/4, column 4(s%4)) and
// output lane i receives k-rows kb..kb+3 of column i.  No transposed copy of
// M is needed.  The tile must hold 32*KW bytes; it is free again on return.
// The layer wavefront's backward loads its weights this way (B = 16: its
// transposes took 18 us per step, the loads add 11; B = 32: 0.803 -> 0.789
// ms).  The per-layer backward keeps a transposed copy: its transpose hides
// behind the exchange fill it carries, while these loads, in 64-byte pieces of
// rows every workgroup of an XCD shares, add 3 us per launch.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

template <int HN, int KW>
__device__ __forceinline__ void load_resident_cols(const bf16_t *M, long ld, long rows, int j0, int k0,
                                                   unsigned tile, const char *tilep, int lane,
                                                   u32x4 (&rf)[HN >= 16 ? HN / 16 : 1][KW / 32])
{
    constexpr int NBB = HN >= 16 ? HN / 16 : 1;
    constexpr int PITCH = 32 * NBB;           // bytes per staged k-row: NC = 16 NBB columns
    constexpr int PR = KW / NBB;              // k-rows per pass
    constexpr int RPI = 1024 / PITCH;         // k-rows per 1 KiB instruction
    constexpr int NI = PR / RPI;              // instructions per pass
    constexpr int CPP = PR / 32;              // 32-deep chunks per pass
    static_assert(PR % RPI == 0 && PR % 32 == 0 && NI >= 1, "whole instructions and chunks per pass");
    const u32x4 rs = buffer_desc(M, rows * ld * 2);
    const int rin = lane / (PITCH / 16), col = (lane % (PITCH / 16)) * 8;
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int p = 0; p < NBB; ++p) {
        if (p > 0) wait_own_lds();   // the previous pass's reads are done before its tile is overwritten
#pragma unroll
        for (int q = 0; q < NI; ++q) {
            const long k = k0 + p * PR + q * RPI + rin;
            const unsigned voff = col < HN ? (unsigned)((k * ld + j0 + col) * 2) : OOB_OFFSET;
            dma16(rs, __builtin_amdgcn_readfirstlane(tile + q * 1024), voff);
        }
        wait_own_loads();
#pragma unroll
        for (int cc = 0; cc < CPP; ++cc) {
            const int c = p * CPP + cc;
#pragma unroll
            for (int i = 0; i < NBB; ++i) {
                const int kb = cc * 32 + g * 8;
                const int off = (kb + s / 4) * PITCH + (16 * i + 4 * (s % 4)) * 2;
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(tilep + off));
                const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(tilep + off + 4 * PITCH));
                const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
                rf[i][c] = (16 * i + s) < HN ? u32x4{l2[0], l2[1], h2[0], h2[1]} : zero16();
            }
        }
    }
    wait_own_lds();
}

// a + b of eight bf16 pairs, in fp32, rounded to bf16 as the element-wise
// add kernel rounds them (a result equal to NOT_READY becomes the canonical
// NaN, as for every exchanged value).
__device__ __forceinline__ u32x4 bf16_add8(u32x4 a, u32x4 b)
{
    u32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float lo = __uint_as_float(a[i] << 16) + __uint_as_float(b[i] << 16);
        const float hi = __uint_as_float(a[i] & 0xffff0000u) + __uint_as_float(b[i] & 0xffff0000u);
        r[i] = (unsigned)ready_value(f32_to_bf16(lo)) | ((unsigned)ready_value(f32_to_bf16(hi)) << 16);
    }
    return r;
}

// The residual form of stage_mma_when_ready: the rows multiplied are the sums
// a + b of two row sets (a residual layer's output y + x), each either
// exchanged (poll_*: copied with loads that miss L1 and repeated while an
// element of a valid row holds NOT_READY) or complete before the launch.
// Once every element is final and `store` is set, the wave also stores its
// slice of the summed rows into `rsum` with device-coherent stores (one
// workgroup per XCD stores them; each element is written once).
template <int RB, int KCW, int NBX>
__device__ __forceinline__ bool stage_sum_mma_when_ready(u32x4 rsa, u32x4 rsb, bool poll_a, bool poll_b, long r0,
                                                         long ld, int kbyte, unsigned tile_a, const char *tpa,
                                                         unsigned tile_b, const char *tpb, int lane, int valid,
                                                         const u32x4 (&rf)[NBX][KCW], f32x4 (&acc)[NBX],
                                                         __amdgpu_buffer_rsrc_t rsum, bool store, unsigned *flags,
                                                         unsigned long long timeout)
{
    constexpr int RPI = 1024 / RB > 0 ? 1024 / RB : 1;
    static_assert(RB <= 1024, "one row per instruction at most");
    const __amdgpu_buffer_rsrc_t rfl = rsrc(flags);
    const bool row_in = (lane & 15) < valid;
    const unsigned long long t0 = wall_clock64();
    unsigned qmask = 0;
#pragma unroll
    for (int q = 0; q < 16 / RPI; ++q)
        if (q * RPI < valid) qmask |= 1u << q;
    while (true) {
        if (poll_a)
            stage_rows<RB, true>(rsa, r0, ld, kbyte, tile_a, lane, qmask);
        else
            stage_rows<RB, false>(rsa, r0, ld, kbyte, tile_a, lane, qmask);
        if (poll_b)
            stage_rows<RB, true>(rsb, r0, ld, kbyte, tile_b, lane, qmask);
        else
            stage_rows<RB, false>(rsb, r0, ld, kbyte, tile_b, lane, qmask);
        const unsigned ab = __builtin_amdgcn_raw_buffer_load_b32(rfl, XCD_ABORT * 4, 0, 16);
        wait_own_loads();
#pragma unroll
        for (int i = 0; i < NBX; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        u16x2 seen = {0, 0};
#pragma unroll
        for (int c = 0; c < KCW; ++c) {
            const u32x4 fa = stage_frag<RB>(tpa, c, lane);
            const u32x4 fb = stage_frag<RB>(tpb, c, lane);
            if (poll_a) seen = max_halves(seen, fa);
            if (poll_b) seen = max_halves(seen, fb);
            const u32x4 fs = bf16_add8(fa, fb);
#pragma unroll
            for (int i = 0; i < NBX; ++i) mfma16(acc[i], rf[i][c], fs, bf16_t{});
        }
        const unsigned long long lm = __builtin_amdgcn_ballot_w64(saw_not_ready(seen) && row_in);
        if (lm == 0) {
            if (store && row_in) {   // lane: row lane % 16, k = c*32 + (lane/16)*8 .. +7 of the wave's slice
#pragma unroll
                for (int c = 0; c < KCW; ++c) {
                    const u32x4 fs = bf16_add8(stage_frag<RB>(tpa, c, lane), stage_frag<RB>(tpb, c, lane));
                    const unsigned off =
                        (unsigned)(((r0 + (lane & 15)) * ld) * 2 + kbyte + c * 64 + (lane >> 4) * 16);
                    __builtin_amdgcn_raw_buffer_store_b128(fs, rsum, off, 0, 16);
                }
            }
            return true;
        }
        if (ab != 0) return false;
        if (wall_clock64() - t0 > timeout) {
            if (lane == 0) {
                __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_WATCHDOG, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(flags + XCD_ABORT, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            return false;
        }
        wait_own_lds();
    }
}

struct XFwdArgs {
    int T, B, H, reverse, RX;
    long ldy;
    const bf16_t *R, *h0;
    const float *c0;
    float *gates, *cs;
    const uint16_t *gx;   // fp16 input projection [T][B][4H] (its bit patterns), or NULL: it is in gates
    f16_t *act;           // fp16 activated gates [T][B][4H] (ACT16), else they go to gates in fp32
    bf16_t *y, *hT;
    float *cT;
    unsigned *flags;
    unsigned long long timeout;
};

// Wave w multiplies the k range [w*H/8, (w+1)*H/8) for all 4*HN gate rows of
// the workgroup's cells; the eight partial sums meet in LDS.  MBX blocks of
// 16 batch rows per XCD.  The resident gate rows are ordered cell-major
// (row 4u + g is gate g of cell u) and the product is taken transposed
// (gate rows x batch rows), so each lane ends with the four gates of one
// cell for one batch row: one 16-byte LDS store per block, and the gate math
// reads each wave's partial sums of a cell with one 16-byte load.
template <int HN, int MBX, bool GX16 = false, bool ACT16 = false>
__global__ __launch_bounds__(XT) void lstm_fwd_xcd(XFwdArgs a)
{
    constexpr int NT = 4 * HN;        // gate rows owned (i, f, g, o of HN cells)
    constexpr int NB = NT / 16;       // 16-row MFMA blocks
    constexpr int KW = 4 * HN;        // k per wave (H / 8)
    constexpr int KCW = KW / 32;      // 32-deep chunks per wave
    constexpr int RB = KW * 2;        // staged bytes per row
    constexpr int NCELL = 16 * HN;    // cells of one row block
    constexpr int RP = NT + 36;       // padded partial-sum row (conflict-free writes, few read conflicts)
    __shared__ __attribute__((aligned(16))) float red[8][16][RP];
    __shared__ __attribute__((aligned(1024))) char stage[8][16 * RB];
    __shared__ int s_xcd;

    if (!claim_role(a.flags, &s_xcd)) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int xcd = s_xcd, slot = blockIdx.x >> 3;
    const int H = a.H, B = a.B;
    const long G4 = 4L * H;
    const int j0 = slot * HN;
    const int row0 = xcd * a.RX, rowend = min(B, row0 + a.RX);
    const unsigned tile = lds_addr(&stage[w][0]);

    // resident weights: the 4*HN rows of R feeding this workgroup's cells
    // (cell-major: row 4u + g), this wave's k range
    u32x4 rf[NB][KCW];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int n = i * 16 + (lane & 15);
        const int g = n & 3, u = n >> 2;
        const bf16_t *rrow = a.R + (long)(g * H + j0 + u) * H + w * KW;
#pragma unroll
        for (int c = 0; c < KCW; ++c) rf[i][c] = ldg16(rrow + c * 32 + (lane >> 4) * 8);
    }
    const u32x4 rs_y = buffer_desc(a.y, (long)a.T * B * a.ldy * 2);
    const u32x4 rs_h0 = buffer_desc(a.h0, (long)B * H * 2);

    const bool has_cell = tid < NCELL;
    const int cr = tid / HN, cu = tid % HN, cj = j0 + cu;
    float creg[MBX];
#pragma unroll
    for (int mb = 0; mb < MBX; ++mb) {
        const int b = row0 + mb * 16 + cr;
        creg[mb] = (has_cell && b < rowend && a.c0) ? a.c0[(long)b * H + cj] : 0.0f;
    }

    __shared__ int s_bad;
    if (tid == 0) s_bad = 0;   // ordered by the first barrier below

    int tprev = 0;
    for (int s = 0; s < a.T; ++s) {
        const int t = a.reverse ? a.T - 1 - s : s;
        const bool last = s == a.T - 1;
        // input projection of this step for the own cells (independent of
        // h_{t-1}), kept as loaded (fp32 or fp16 bits) until the gate math so
        // that no wait for these loads lands before the exchange
        unsigned gxu[MBX][4];
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const int b = row0 + mb * 16 + cr;
            const bool v = has_cell && b < rowend;
            const long e = ((long)t * B + b) * G4 + cj;
            if constexpr (GX16) {
#pragma unroll
                for (int g = 0; g < 4; ++g) gxu[mb][g] = v ? (unsigned)a.gx[e + g * H] : 0u;
            } else {
#pragma unroll
                for (int g = 0; g < 4; ++g) gxu[mb][g] = v ? __float_as_uint(a.gates[e + g * H]) : 0u;
            }
        }
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            f32x4 acc[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int rb0 = row0 + mb * 16;
            if (mb > 0) wait_own_lds();   // the previous block's fragment reads are done
            if (s > 0) {
                if (!stage_mma_when_ready<RB, KCW, NB, true>(rs_y, (long)tprev * B + rb0, a.ldy, w * KW * 2, tile,
                                                             stage[w], lane, rowend - rb0, rf, acc, a.flags, a.timeout,
                                                             slot))
                    s_bad = 1;
            } else if (a.h0) {
                stage_rows<RB>(rs_h0, rb0, H, w * KW * 2, tile, lane);
                wait_own_loads();
#pragma unroll
                for (int c = 0; c < KCW; ++c) {
                    const u32x4 fa = stage_frag<RB>(stage[w], c, lane);
#pragma unroll
                    for (int i = 0; i < NB; ++i) mfma16(acc[i], rf[i][c], fa, bf16_t{});
                }
            }
            // lane: batch row lane%16, gates 0..3 of cell 4i + lane/16 of block i
#pragma unroll
            for (int i = 0; i < NB; ++i)
                *reinterpret_cast<f32x4 *>(&red[w][lane & 15][i * 16 + 4 * (lane >> 4)]) = acc[i];
            __syncthreads();
            if (s_bad) return;   // the same decision in every wave
            // Every lane applies the cell equations (a lane without a cell reads
            // row 0 of the partial sums; lanes without a cell or row produce
            // values nobody stores) and only the stores depend on the lane:
            // the input projection loaded for this step is then consumed on
            // every path, and the next step's loads do not wait for these
            // loads, nor for the stores issued after them.  With four row
            // blocks the registers run short and the lanes without a row skip it.
            constexpr bool ALL_LANES = MBX <= 2;
            const int b = rb0 + cr;
            const int crr = has_cell ? cr : 0;
            if (ALL_LANES || (has_cell && b < rowend)) {
                float z[4];
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    unsigned u = gxu[mb][g];
                    if constexpr (GX16) {
                        // the conversion stays here: hoisted next to its load it
                        // would make that load's wait a full memory latency
                        asm volatile("" : "+v"(u));
                        z[g] = to_f32(__builtin_bit_cast(f16_t, (uint16_t)u));
                    } else {
                        z[g] = __uint_as_float(u);
                    }
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const f32x4 p = *reinterpret_cast<const f32x4 *>(&red[q][crr][4 * cu]);
#pragma unroll
                    for (int g = 0; g < 4; ++g) z[g] += p[g];
                }
                const float ig = sigmoid_f(z[0]), fg = sigmoid_f(z[1]), gg = tanh_f(z[2]), og = sigmoid_f(z[3]);
                const float c = fg * creg[mb] + ig * gg;
                const float m = og * tanh_f(c);
                creg[mb] = c;
                if (has_cell && b < rowend) {
                    const bf16_t hv = ready_value(f32_to_bf16(m));
                    a.y[((long)t * B + b) * a.ldy + cj] = hv;
                    if (last && a.hT) a.hT[(long)b * H + cj] = hv;
                    // saved activations for the backward pass (not on the critical path)
                    if constexpr (ACT16) {
                        f16_t *ap = a.act + ((long)t * B + b) * G4 + cj;
                        ap[0] = (f16_t)ig;
                        ap[H] = (f16_t)fg;
                        ap[2 * H] = (f16_t)gg;
                        ap[3 * H] = (f16_t)og;
                    } else {
                        float *gp = a.gates + ((long)t * B + b) * G4 + cj;
                        gp[0] = ig;
                        gp[H] = fg;
                        gp[2 * H] = gg;
                        gp[3 * H] = og;
                    }
                    a.cs[((long)t * B + b) * H + cj] = c;
                    if (last && a.cT) a.cT[(long)b * H + cj] = c;
                }
            }
            __syncthreads();   // red is rewritten by the next row block or step
        }
        tprev = t;
    }
}

// ---------------------------------------------------------------------------
// Layer wavefront: the forward pass of a stack of L (2..4) unidirectional
// layers in one launch, for batches of at most 32 rows (all rows in one
// XCD).  XCD 2l runs layer l's recurrence with the rows of R_l resident, as
// lstm_fwd_xcd does with all rows in one XCD; XCD 2l+1 (l >= 1) keeps the
// rows of W_l resident and computes each step's input projection y_{l-1,t}
// W_l^T + b_l as soon as layer l-1 has produced y_{l-1,t}.  The layers thus
// advance together, a few steps apart, instead of one after another (the
// pipelining of layers over time steps that model parallelism exploits).
// Rows that cross XCDs (y into the next layer's projection, the projection
// into the recurrence) are stored with device-coherent (sc1) stores and read
// with sc1 loads under the NOT_READY protocol: y is filled with the bf16
// pattern, the projections of layers >= 1 with the fp32 pattern 0xffffffff,
// before the launch.  Layer 0's projection is either given (computed by the
// GEMM before the launch) or computed on XCD 1 from the stack's input x when
// its width is H (x is complete at the launch, so it is read without the
// protocol).
struct WaveLayer {
    const bf16_t *R, *W;
    const float *bias;
    float *gates, *cs;   // gates: the input projection in, the activations out
    bf16_t *y;           // [T][B][H]
    // residual input (the layer below adds its own input to its output): the
    // projection multiplies y of the layer below plus in_b, and stores that
    // sum into `sum`; poll_b: in_b is written in the launch
    const bf16_t *in_b;
    bf16_t *sum;
    int poll_b;
};

struct XWaveArgs {
    int T, B, H, L;
    const bf16_t *x;     // the stack's input [T][B][H] when XCD 1 projects it; NULL: layer 0's projection is given
    WaveLayer ly[4];
    unsigned *flags;
    unsigned long long timeout;
};

constexpr unsigned NOT_READY_F32 = 0xffffffffu;

__device__ __forceinline__ unsigned ready_f32(float v)
{
    const unsigned u = __float_as_uint(v);
    return u == NOT_READY_F32 ? 0x7fc00000u : u;
}

template <int HN, int MBX, bool RES = false>
__global__ __launch_bounds__(XT) void lstm_fwd_wave(XWaveArgs a)
{
    constexpr int NT = 4 * HN;        // gate rows owned (i, f, g, o of HN cells)
    constexpr int NB = NT / 16;
    constexpr int KW = 4 * HN;        // k per wave (H / 8)
    constexpr int KCW = KW / 32;
    constexpr int RB = KW * 2;
    constexpr int NCELL = 16 * HN;
    constexpr int RP = NT + 36;
    __shared__ __attribute__((aligned(16))) float red[8][16][RP];
    __shared__ __attribute__((aligned(1024))) char stage[8][16 * RB];
    __shared__ __attribute__((aligned(1024))) char stage_b[RES ? 8 : 1][RES ? 16 * RB : 16];   // second addend
    __shared__ int s_xcd;
    __shared__ int s_bad;

    if (!claim_role(a.flags, &s_xcd)) return;
    const int xcd = s_xcd, layer = xcd >> 1;
    const bool wrole = (xcd & 1) != 0;
    if (layer >= a.L || (wrole && layer == 0 && !a.x)) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, slot = blockIdx.x >> 3;
    const int H = a.H, B = a.B;
    const long G4 = 4L * H;
    const int j0 = slot * HN;
    const unsigned tile = lds_addr(&stage[w][0]);
    const WaveLayer ly = a.ly[layer];

    // resident weights: the 4*HN rows of R_l (recurrence) or W_l (projection)
    // feeding the owned cells, cell-major (row 4u + g), this wave's k range
    const bf16_t *M = wrole ? ly.W : ly.R;
    u32x4 rf[NB][KCW];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int n = i * 16 + (lane & 15);
        const int g = n & 3, u = n >> 2;
        const bf16_t *rrow = M + (long)(g * H + j0 + u) * H + w * KW;
#pragma unroll
        for (int c = 0; c < KCW; ++c) rf[i][c] = ldg16(rrow + c * 32 + (lane >> 4) * 8);
    }
    const bool has_cell = tid < NCELL;
    const int cr = tid / HN, cu = tid % HN, cj = j0 + cu;
    const int crr = has_cell ? cr : 0;
    // bounded descriptors: lanes without a row read rows past the last step
    // at the end (those loads return zero), and no store leaves its tensor
    const __amdgpu_buffer_rsrc_t rg =
        __builtin_amdgcn_make_buffer_rsrc(ly.gates, (short)0, (int)((long)a.T * B * G4 * 4), 0x00020000);
    if (tid == 0) s_bad = 0;   // ordered by the first barrier below

    if (wrole) {
        // input projection of layer l from the rows of y_{l-1} (of x for layer 0)
        const bool from_x = layer == 0;
        const u32x4 rs_x = buffer_desc(from_x ? a.x : a.ly[layer - 1].y, (long)a.T * B * H * 2);
        float bz[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) bz[g] = has_cell ? ly.bias[g * H + cj] : 0.0f;
        for (int s = 0; s < a.T; ++s) {
#pragma unroll
            for (int mb = 0; mb < MBX; ++mb) {
                const int rb0 = mb * 16;
                f32x4 acc[NB];
#pragma unroll
                for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (from_x) {
                    if (s > 0 || mb > 0) wait_own_lds();   // the previous block's fragment reads are done
                    stage_rows<RB>(rs_x, (long)s * B + rb0, H, w * KW * 2, tile, lane);
                    wait_own_loads();
#pragma unroll
                    for (int c = 0; c < KCW; ++c) {
                        const u32x4 fa = stage_frag<RB>(stage[w], c, lane);
#pragma unroll
                        for (int i = 0; i < NB; ++i) mfma16(acc[i], rf[i][c], fa, bf16_t{});
                    }
                } else if (RES && ly.in_b) {   // the layer below is residual: multiply y + its input
                    if (mb > 0) wait_own_lds();
                    const u32x4 rs_b = buffer_desc(ly.in_b, (long)a.T * B * H * 2);
                    const __amdgpu_buffer_rsrc_t rsum =
                        __builtin_amdgcn_make_buffer_rsrc(ly.sum, (short)0, (int)((long)a.T * B * H * 2), 0x00020000);
                    if (!stage_sum_mma_when_ready<RB, KCW, NB>(rs_x, rs_b, true, ly.poll_b != 0, (long)s * B + rb0, H,
                                                               w * KW * 2, tile, stage[w],
                                                               lds_addr(&stage_b[RES ? w : 0][0]),
                                                               stage_b[RES ? w : 0], lane, B - rb0, rf, acc, rsum,
                                                               slot == 0, a.flags, a.timeout))
                        s_bad = 1;
                } else {
                    if (mb > 0) wait_own_lds();
                    if (!stage_mma_when_ready<RB, KCW, NB, true>(rs_x, (long)s * B + rb0, H, w * KW * 2, tile,
                                                                 stage[w], lane, B - rb0, rf, acc, a.flags, a.timeout,
                                                                 slot))
                        s_bad = 1;
                }
#pragma unroll
                for (int i = 0; i < NB; ++i)
                    *reinterpret_cast<f32x4 *>(&red[w][lane & 15][i * 16 + 4 * (lane >> 4)]) = acc[i];
                __syncthreads();
                if (s_bad) return;
                if (has_cell && rb0 + cr < B) {
                    float z[4] = {bz[0], bz[1], bz[2], bz[3]};
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        const f32x4 p = *reinterpret_cast<const f32x4 *>(&red[q][cr][4 * cu]);
#pragma unroll
                        for (int g = 0; g < 4; ++g) z[g] += p[g];
                    }
                    const unsigned off = (unsigned)((((long)s * B + rb0 + cr) * G4 + cj) * 4);
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        __builtin_amdgcn_raw_buffer_store_b32(ready_f32(z[g]), rg, off + (unsigned)(g * H * 4), 0, 16);
                }
                __syncthreads();   // red is rewritten by the next block or step
            }
        }
        return;
    }

    // recurrence of layer l
    const u32x4 rs_y = buffer_desc(ly.y, (long)a.T * B * H * 2);
    const __amdgpu_buffer_rsrc_t ryw =
        __builtin_amdgcn_make_buffer_rsrc(ly.y, (short)0, (int)((long)a.T * B * H * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t rfl = rsrc(a.flags);
    const bool poll_gx = layer > 0 || a.x != nullptr;
    float creg[MBX];
#pragma unroll
    for (int mb = 0; mb < MBX; ++mb) creg[mb] = 0.0f;
    for (int s = 0; s < a.T; ++s) {
        // this step's input projection (may still be in flight when computed in the launch)
        unsigned gxu[MBX][4];
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const unsigned goff = (unsigned)((((long)s * B + mb * 16 + crr) * G4 + cj) * 4);
#pragma unroll
            for (int g = 0; g < 4; ++g)
                gxu[mb][g] = poll_gx ? __builtin_amdgcn_raw_buffer_load_b32(rg, goff + (unsigned)(g * H * 4), 0, 16)
                                     : __builtin_amdgcn_raw_buffer_load_b32(rg, goff + (unsigned)(g * H * 4), 0, 0);
        }
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const int rb0 = mb * 16;
            const bool vrow = has_cell && rb0 + cr < B;
            f32x4 acc[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (mb > 0) wait_own_lds();   // the previous block's fragment reads are done
            if (s > 0) {
                if (!stage_mma_when_ready<RB, KCW, NB, true>(rs_y, (long)(s - 1) * B + rb0, H, w * KW * 2, tile,
                                                             stage[w], lane, B - rb0, rf, acc, a.flags, a.timeout,
                                                             slot))
                    s_bad = 1;
            }
#pragma unroll
            for (int i = 0; i < NB; ++i)
                *reinterpret_cast<f32x4 *>(&red[w][lane & 15][i * 16 + 4 * (lane >> 4)]) = acc[i];
            __syncthreads();
            if (s_bad) return;
            if (poll_gx) {   // re-read the elements that still hold NOT_READY
                const unsigned goff = (unsigned)((((long)s * B + rb0 + crr) * G4 + cj) * 4);
                const unsigned long long t0 = wall_clock64();
                while (true) {
                    bool nr = false;
#pragma unroll
                    for (int g = 0; g < 4; ++g) nr = nr || (vrow && gxu[mb][g] == NOT_READY_F32);
                    if (__builtin_amdgcn_ballot_w64(nr) == 0) break;
                    const unsigned ab = __builtin_amdgcn_raw_buffer_load_b32(rfl, XCD_ABORT * 4, 0, 16);
                    if (ab != 0 || wall_clock64() - t0 > a.timeout) {
                        if (lane == 0 && ab == 0) {
                            __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_WATCHDOG, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                            __hip_atomic_store(a.flags + XCD_ABORT, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        }
                        s_bad = 1;
                        break;
                    }
                    for (int g = 0; g < 4; ++g)
                        if (vrow && gxu[mb][g] == NOT_READY_F32)
                            gxu[mb][g] = __builtin_amdgcn_raw_buffer_load_b32(rg, goff + (unsigned)(g * H * 4), 0, 16);
                }
            }
            {
                float z[4];
#pragma unroll
                for (int g = 0; g < 4; ++g) z[g] = __uint_as_float(gxu[mb][g]);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const f32x4 p = *reinterpret_cast<const f32x4 *>(&red[q][crr][4 * cu]);
#pragma unroll
                    for (int g = 0; g < 4; ++g) z[g] += p[g];
                }
                const float ig = sigmoid_f(z[0]), fg = sigmoid_f(z[1]), gg = tanh_f(z[2]), og = sigmoid_f(z[3]);
                const float c = fg * creg[mb] + ig * gg;
                const float m = og * tanh_f(c);
                creg[mb] = c;
                if (vrow) {
                    const long row = (long)s * B + rb0 + cr;
                    const bf16_t hv = ready_value(f32_to_bf16(m));
                    __builtin_amdgcn_raw_buffer_store_b16(hv, ryw, (unsigned)((row * H + cj) * 2), 0, 16);
                    // saved activations for the backward pass (not on the critical path)
                    float *gp = ly.gates + row * G4 + cj;
                    gp[0] = ig;
                    gp[H] = fg;
                    gp[2 * H] = gg;
                    gp[3 * H] = og;
                    ly.cs[row * H + cj] = c;
                }
            }
            __syncthreads();   // red is rewritten by the next block or step
            if (s_bad) return;
        }
    }
}

// Backward of the layer wavefront (stacks of 2..4 layers with I = H = 1024,
// at most 32 batch rows): XCD 2l runs layer l's BPTT with the rows of R_l^T
// resident and stores dz_l; XCD 2l+1 multiplies each step's dz_{l,t} by W_l
// (the rows of W_l^T resident) into dx_{l,t}, which is the upstream gradient
// dy_{l-1,t} of layer l-1 (for l = 0 the stack's input gradient).  Layer
// l-1's BPTT thus follows layer l's a few steps behind.  dz and the dy rows
// that cross XCDs are stored with sc1 stores and read with sc1 loads under
// the NOT_READY protocol (both filled before the launch).
struct WaveBwdLayer {
    const bf16_t *R, *W;       // [4H][H]: R_l, W_l (W NULL: no input gradient wanted)
    const float *gates, *cs;   // activations and cell states saved by the forward
    bf16_t *dz;                // [T][B][4H]
    const bf16_t *dy;          // [T][B][H] upstream gradient (for l < L-1 written by XCD 2l+3)
    bf16_t *dx;                // [T][B][H] input gradient (dy of layer l-1, or the stack's dx)
    float *dbp;                // [4H] bias gradient of layer l
};

struct XWaveBwdArgs {
    int T, B, H, L;
    WaveBwdLayer ly[4];
    unsigned *flags;
    unsigned long long timeout;
    int res_mask;   // bit l: layer l is residual, its dy also reaches its dx unchanged
};

template <int HN, int MBX, bool RES = false>
__global__ __launch_bounds__(XT) void lstm_bwd_wave(XWaveBwdArgs a)
{
    constexpr int NBB = HN / 16;
    constexpr int NC = 16 * NBB;
    constexpr int KW = 16 * HN;                   // k per wave (4H / 8)
    constexpr int KCW = KW / 32;
    constexpr int RB = KW * 2;
    constexpr int NCELL = 16 * HN;
    constexpr int RP = NC + 4;
    __shared__ float red[8][16][RP];
    __shared__ __attribute__((aligned(1024))) char stage[8][16 * RB];
    __shared__ int s_xcd;
    __shared__ int s_bad;

    if (!claim_role(a.flags, &s_xcd)) return;
    const int xcd = s_xcd, layer = xcd >> 1;
    const bool xrole = (xcd & 1) != 0;
    if (layer >= a.L) return;
    const WaveBwdLayer ly = a.ly[layer];
    if (xrole && !ly.W) return;
    const bool lres = RES && ((a.res_mask >> layer) & 1);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, slot = blockIdx.x >> 3;
    const int H = a.H, B = a.B, T = a.T;
    const long G4 = 4L * H;
    const int j0 = slot * HN;
    const unsigned tile = lds_addr(&stage[w][0]);

    // resident: columns j0.. of R_l (BPTT) or W_l (input gradient), this wave's k range
    u32x4 rf[NBB][KCW];
    load_resident_cols<HN, KW>(xrole ? ly.W : ly.R, H, G4, j0, w * KW, tile, stage[w], lane, rf);
    const u32x4 rs_dz = buffer_desc(ly.dz, (long)T * B * G4 * 2);
    const bool has_cell = tid < NCELL;
    const int cr = tid / HN, cu = tid % HN, cj = j0 + cu;
    const int crr = has_cell ? cr : 0;
    if (tid == 0) s_bad = 0;   // ordered by the first barrier below

    if (xrole) {
        const __amdgpu_buffer_rsrc_t rdx =
            __builtin_amdgcn_make_buffer_rsrc(ly.dx, (short)0, (int)((long)T * B * H * 2), 0x00020000);
        for (int s = T - 1; s >= 0; --s) {
#pragma unroll
            for (int mb = 0; mb < MBX; ++mb) {
                const int rb0 = mb * 16;
                f32x4 acc[NBB];
#pragma unroll
                for (int i = 0; i < NBB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (mb > 0) wait_own_lds();
                if (!stage_mma_when_ready<RB, KCW, NBB>(rs_dz, (long)s * B + rb0, G4, w * KW * 2, tile, stage[w], lane,
                                                        B - rb0, rf, acc, a.flags, a.timeout, slot))
                    s_bad = 1;
#pragma unroll
                for (int i = 0; i < NBB; ++i)
#pragma unroll
                    for (int v = 0; v < 4; ++v) red[w][4 * (lane >> 4) + v][i * 16 + (lane & 15)] = acc[i][v];
                __syncthreads();
                if (s_bad) return;
                const bool vr = has_cell && rb0 + cr < B;
                // residual layer: its upstream gradient also reaches its input unchanged
                // (written in the launch by the layer above, except for the top layer)
                bf16_t g = 0;
                if (RES && lres) {
                    const bool poll_res = layer < a.L - 1;
                    const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
                        const_cast<bf16_t *>(ly.dy), (short)0, (int)((long)T * B * H * 2), 0x00020000);
                    const unsigned off = (unsigned)((((long)s * B + rb0 + crr) * H + cj) * 2);
                    if (vr)   // sc1 (16): the rows written in the launch are read past L1
                        g = poll_res ? (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(rres, off, 0, 16)
                                     : (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(rres, off, 0, 0);
                    if (poll_res) {
                        const __amdgpu_buffer_rsrc_t rfl = rsrc(a.flags);
                        const unsigned long long t0 = wall_clock64();
                        while (__builtin_amdgcn_ballot_w64(vr && g == NOT_READY) != 0) {
                            const unsigned ab = __builtin_amdgcn_raw_buffer_load_b32(rfl, XCD_ABORT * 4, 0, 16);
                            if (ab != 0 || wall_clock64() - t0 > a.timeout) {
                                if (lane == 0 && ab == 0) {
                                    __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_WATCHDOG, __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_AGENT);
                                    __hip_atomic_store(a.flags + XCD_ABORT, 1u, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                                }
                                s_bad = 1;
                                break;
                            }
                            if (vr && g == NOT_READY) g = (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(rres, off, 0, 16);
                        }
                    }
                }
                if (vr) {
                    float v = 0.0f;
#pragma unroll
                    for (int q = 0; q < 8; ++q) v += red[q][cr][cu];
                    if (RES && lres) v += to_f32(g);
                    __builtin_amdgcn_raw_buffer_store_b16(ready_value(f32_to_bf16(v)), rdx,
                                                          (unsigned)((((long)s * B + rb0 + cr) * H + cj) * 2), 0, 16);
                }
                __syncthreads();   // red is rewritten by the next block or step
                if (RES && s_bad) return;
            }
        }
        return;
    }

    // BPTT of layer l
    const __amdgpu_buffer_rsrc_t rdzw =
        __builtin_amdgcn_make_buffer_rsrc(ly.dz, (short)0, (int)((long)T * B * G4 * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t rdy =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t *>(ly.dy), (short)0, (int)((long)T * B * H * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t rfl = rsrc(a.flags);
    const bool poll_dy = layer < a.L - 1;
    float dhn[MBX], dcn[MBX];
    float dbacc[4] = {0.f, 0.f, 0.f, 0.f};
    bf16_t dyv[MBX];
    float gv[MBX][4], cv[MBX], cpv[MBX];
#pragma unroll
    for (int mb = 0; mb < MBX; ++mb) dhn[mb] = dcn[mb] = 0.0f;
    auto load_inputs = [&](int s) {
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const bool v = has_cell && mb * 16 + cr < B;
            const unsigned doff = (unsigned)((((long)s * B + mb * 16 + crr) * H + cj) * 2);
            dyv[mb] = poll_dy ? (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(rdy, doff, 0, 16)
                              : (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(rdy, doff, 0, 0);
            const long rt = (long)s * B + (v ? mb * 16 + cr : 0);
#pragma unroll
            for (int g = 0; g < 4; ++g) gv[mb][g] = v ? ly.gates[rt * G4 + g * H + cj] : 0.0f;
            cv[mb] = v ? ly.cs[rt * H + cj] : 0.0f;
            cpv[mb] = (v && s > 0) ? ly.cs[(rt - B) * H + cj] : 0.0f;
        }
    };
    load_inputs(T - 1);
    for (int s = T - 1; s >= 0; --s) {
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const bool vrow = has_cell && mb * 16 + cr < B;
            if (poll_dy) {   // the upstream gradient of this step may still be in flight
                const unsigned doff = (unsigned)((((long)s * B + mb * 16 + crr) * H + cj) * 2);
                const unsigned long long t0 = wall_clock64();
                while (__builtin_amdgcn_ballot_w64(vrow && dyv[mb] == NOT_READY) != 0) {
                    const unsigned ab = __builtin_amdgcn_raw_buffer_load_b32(rfl, XCD_ABORT * 4, 0, 16);
                    if (ab != 0 || wall_clock64() - t0 > a.timeout) {
                        if (lane == 0 && ab == 0) {
                            __hip_atomic_fetch_or(&g_xcd_tripped, TRIP_WATCHDOG, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                            __hip_atomic_store(a.flags + XCD_ABORT, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        }
                        s_bad = 1;
                        break;
                    }
                    if (vrow && dyv[mb] == NOT_READY)
                        dyv[mb] = (bf16_t)__builtin_amdgcn_raw_buffer_load_b16(rdy, doff, 0, 16);
                }
            }
            // gate gradients of the owned cells (every lane computes, only the stores depend on the lane)
            const float ig = gv[mb][0], fg = gv[mb][1], gg = gv[mb][2], og = gv[mb][3];
            const float dm = to_f32(dyv[mb]) + dhn[mb];
            const float tc = tanh_f(cv[mb]);
            const float d_o = dm * tc;
            const float d_c = dcn[mb] + dm * og * (1.0f - tc * tc);
            const float d_i = d_c * gg, d_g = d_c * ig, d_f = d_c * cpv[mb];
            const float z[4] = {d_i * ig * (1.0f - ig), d_f * fg * (1.0f - fg), d_g * (1.0f - gg * gg),
                                d_o * og * (1.0f - og)};
            if (vrow) {
                const unsigned zoff = (unsigned)((((long)s * B + mb * 16 + cr) * G4 + cj) * 2);
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    __builtin_amdgcn_raw_buffer_store_b16(ready_value(f32_to_bf16(z[g])), rdzw,
                                                          zoff + (unsigned)(g * H * 2), 0, 16);
            }
#pragma unroll
            for (int g = 0; g < 4; ++g) dbacc[g] += vrow ? z[g] : 0.0f;
            dcn[mb] = d_c * fg;
        }
        if (s == 0) break;
        load_inputs(s - 1);
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const int rb0 = mb * 16;
            f32x4 acc[NBB];
#pragma unroll
            for (int i = 0; i < NBB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (mb > 0) wait_own_lds();
            if (!stage_mma_when_ready<RB, KCW, NBB>(rs_dz, (long)s * B + rb0, G4, w * KW * 2, tile, stage[w], lane,
                                                    B - rb0, rf, acc, a.flags, a.timeout, slot))
                s_bad = 1;
#pragma unroll
            for (int i = 0; i < NBB; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) red[w][4 * (lane >> 4) + v][i * 16 + (lane & 15)] = acc[i][v];
            __syncthreads();
            if (s_bad) return;
            if (has_cell && rb0 + cr < B) {
                float v = 0.0f;
#pragma unroll
                for (int q = 0; q < 8; ++q) v += red[q][cr][cu];
                dhn[mb] = v;
            }
            __syncthreads();
        }
    }
    // bias gradient of layer l: sum this workgroup's rows (in row order)
    {
        float *dred = &red[0][0][0];                  // 16 x HN x 4 floats fit in red
        __syncthreads();
        if (has_cell) {
#pragma unroll
            for (int g = 0; g < 4; ++g) dred[(cr * HN + cu) * 4 + g] = dbacc[g];
        }
        __syncthreads();
        if (tid < 4 * HN) {
            const int g = tid / HN, u = tid % HN;
            float v = 0.0f;
            for (int r = 0; r < 16; ++r) v += dred[(r * HN + u) * 4 + g];
            ly.dbp[g * H + j0 + u] = v;
        }
    }
}

struct XBwdArgs {
    int T, B, H, reverse, RX;
    long ldy;
    const bf16_t *Rt, *dy, *dhT;
    const float *dcT, *c0, *gates, *cs;
    const uint16_t *act;   // fp16 activated gates [T][B][4H] (ACT16), else they are in gates
    bf16_t *dz, *dh0;
    float *dc0;
    float *dbpart;          // [8][4H]: per-XCD sums over its rows and all steps of dz
    unsigned *flags;
    unsigned long long timeout;
};

// Per-cell inputs of one BPTT step (saved forward state and upstream gradient).
// dy and fp16 activations stay in their storage bits until they are used:
// converting them where they are loaded would make the wave wait for those
// loads, and with them for the dz stores issued before, ahead of the
// exchange copy.
template <int MBX, bool ACT16>
struct BwdIn {
    bf16_t dy[MBX];
    typename std::conditional<ACT16, unsigned, float>::type g[MBX][4];   // fp16 bit patterns or fp32
    float c[MBX], cp[MBX];
};

// Four fp16 activations from their bit patterns, converted where they are
// used (the empty asm keeps the conversion from moving up to the load).
__device__ __forceinline__ void act_f32(const unsigned (&bits)[4], float (&v)[4])
{
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        unsigned u = bits[g];
        asm volatile("" : "+v"(u));
        v[g] = to_f32(__builtin_bit_cast(f16_t, (uint16_t)u));
    }
}

// Wave w multiplies the k range [w*H/2, (w+1)*H/2) of dh_{t-1} = R^T dz_t
// (k over the 4H gate rows); the eight partial sums meet in LDS.
template <int HN, int MBX, bool ACT16 = false>
__global__ __launch_bounds__(XT) void lstm_bwd_xcd(XBwdArgs a)
{
    constexpr int NBB = HN >= 16 ? HN / 16 : 1;   // 16-column blocks of owned cells
    constexpr int NC = 16 * NBB;
    constexpr int KW = 16 * HN;                   // k per wave (4H / 8)
    constexpr int KCW = KW / 32;
    constexpr int RB = KW * 2;
    constexpr int NCELL = 16 * HN;
    constexpr int RP = NC + 4;                    // padded partial-sum row (conflict-free writes)
    __shared__ float red[8][16][RP];
    __shared__ __attribute__((aligned(1024))) char stage[8][16 * RB];
    __shared__ int s_xcd;

    if (!claim_role(a.flags, &s_xcd)) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int xcd = s_xcd, slot = blockIdx.x >> 3;
    const int H = a.H, B = a.B;
    const long G4 = 4L * H;
    const int j0 = slot * HN;
    const int row0 = xcd * a.RX, rowend = min(B, row0 + a.RX);
    const unsigned tile = lds_addr(&stage[w][0]);

    // resident weights: rows of R^T (= columns of R) of the owned cells, this wave's k range
    u32x4 rf[NBB][KCW];
#pragma unroll
    for (int i = 0; i < NBB; ++i) {
        const int n = i * 16 + (lane & 15);
        const bf16_t *rrow = a.Rt + (long)(j0 + (n < HN ? n : 0)) * G4 + w * KW;
#pragma unroll
        for (int c = 0; c < KCW; ++c) rf[i][c] = n < HN ? ldg16(rrow + c * 32 + (lane >> 4) * 8) : zero16();
    }
    const u32x4 rs_dz = buffer_desc(a.dz, (long)a.T * B * G4 * 2);

    const bool has_cell = tid < NCELL;
    const int cr = tid / HN, cu = tid % HN, cj = j0 + cu;
    auto load_inputs = [&](int s, BwdIn<MBX, ACT16> &in) {
        const int t = a.reverse ? a.T - 1 - s : s;
        const int tp = a.reverse ? t + 1 : t - 1;
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const int b = row0 + mb * 16 + cr;
            const bool v = has_cell && b < rowend;
            const long rt = (long)t * B + (v ? b : 0);
            in.dy[mb] = v ? a.dy[rt * a.ldy + cj] : (bf16_t)0;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                if constexpr (ACT16)
                    in.g[mb][g] = v ? (unsigned)a.act[rt * G4 + g * H + cj] : 0u;
                else
                    in.g[mb][g] = v ? a.gates[rt * G4 + g * H + cj] : 0.0f;
            }
            in.c[mb] = v ? a.cs[rt * H + cj] : 0.0f;
            in.cp[mb] = (v && s > 0) ? a.cs[((long)tp * B + b) * H + cj]
                                     : ((v && a.c0) ? a.c0[(long)(v ? b : 0) * H + cj] : 0.0f);
        }
    };

    float dhn[MBX], dcn[MBX];
    float dbacc[4] = {0.f, 0.f, 0.f, 0.f};   // this thread's rows, summed over steps
#pragma unroll
    for (int mb = 0; mb < MBX; ++mb) {
        const int b = row0 + mb * 16 + cr;
        const bool v = has_cell && b < rowend;
        dhn[mb] = (v && a.dhT) ? to_f32(a.dhT[(long)b * H + cj]) : 0.0f;
        dcn[mb] = (v && a.dcT) ? a.dcT[(long)b * H + cj] : 0.0f;
    }
    BwdIn<MBX, ACT16> in;
    load_inputs(a.T - 1, in);
    __shared__ int s_bad;
    if (tid == 0) s_bad = 0;   // ordered by the first barrier below

    for (int s = a.T - 1; s >= 0; --s) {
        const int t = a.reverse ? a.T - 1 - s : s;
        // gate gradients of the owned cells.  Every lane computes them (lanes
        // without a cell or row loaded zeros) and only the stores depend on
        // the lane: each prefetched input is then consumed on every path, and
        // the next prefetch does not wait for the previous one (nor for the
        // dz stores issued after it) before the exchange copy.  With four row
        // blocks the registers run short and the lanes without a row skip it.
        constexpr bool ALL_LANES = MBX <= 2;
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const int b = row0 + mb * 16 + cr;
            const bool v = has_cell && b < rowend;
            if (!ALL_LANES && !v) continue;
            float gv[4];
            if constexpr (ACT16) {
                act_f32(in.g[mb], gv);
            } else {
#pragma unroll
                for (int g = 0; g < 4; ++g) gv[g] = in.g[mb][g];
            }
            const float ig = gv[0], fg = gv[1], gg = gv[2], og = gv[3];
            const float dm = to_f32(in.dy[mb]) + dhn[mb];
            const float tc = tanh_f(in.c[mb]);
            const float d_o = dm * tc;
            const float d_c = dcn[mb] + dm * og * (1.0f - tc * tc);
            const float d_i = d_c * gg, d_g = d_c * ig, d_f = d_c * in.cp[mb];
            const float zi = d_i * ig * (1.0f - ig), zf = d_f * fg * (1.0f - fg);
            const float zg = d_g * (1.0f - gg * gg), zo = d_o * og * (1.0f - og);
            if (v) {
                bf16_t *dzp = a.dz + ((long)t * B + b) * G4 + cj;
                dzp[0] = ready_value(f32_to_bf16(zi));
                dzp[H] = ready_value(f32_to_bf16(zf));
                dzp[2 * H] = ready_value(f32_to_bf16(zg));
                dzp[3 * H] = ready_value(f32_to_bf16(zo));
            }
            dbacc[0] += v ? zi : 0.0f;
            dbacc[1] += v ? zf : 0.0f;
            dbacc[2] += v ? zg : 0.0f;
            dbacc[3] += v ? zo : 0.0f;
            dcn[mb] = d_c * fg;
            if (v && s == 0 && a.dc0) a.dc0[(long)b * H + cj] = dcn[mb];
        }
        if (s == 0 && !a.dh0) break;
        // the next step's inputs travel while this step's dz is exchanged
        if (s > 0) load_inputs(s - 1, in);
        // dh_{t-1} for the owned cells: dz_t of this XCD's rows times the resident R^T rows
#pragma unroll
        for (int mb = 0; mb < MBX; ++mb) {
            const int rb0 = row0 + mb * 16;
            if (mb > 0) wait_own_lds();
            f32x4 acc[NBB];
#pragma unroll
            for (int i = 0; i < NBB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (!stage_dz<RB, KCW, NBB, MBX>(rs_dz, (long)t * B + rb0, G4, w * KW * 2, tile, stage[w], lane,
                                             rowend - rb0, rf, acc, a.flags, a.timeout, slot))
                s_bad = 1;
#pragma unroll
            for (int i = 0; i < NBB; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) red[w][4 * (lane >> 4) + v][i * 16 + (lane & 15)] = acc[i][v];
            __syncthreads();
            if (s_bad) return;   // the same decision in every wave
            const int bc = rb0 + cr;
            if (has_cell && bc < rowend) {
                float v = 0.0f;
#pragma unroll
                for (int q = 0; q < 8; ++q) v += red[q][cr][cu];
                if (s > 0)
                    dhn[mb] = v;
                else
                    a.dh0[(long)bc * H + cj] = f32_to_bf16(v);
            }
            __syncthreads();
        }
    }
    // bias gradient: sum this workgroup's rows (in row order), one partial per XCD
    {
        float *dred = &red[0][0][0];                  // 16 x HN x 4 floats fit in red
        __syncthreads();
        if (has_cell) {
#pragma unroll
            for (int g = 0; g < 4; ++g) dred[(cr * HN + cu) * 4 + g] = dbacc[g];
        }
        __syncthreads();
        if (tid < 4 * HN) {
            const int g = tid / HN, u = tid % HN;
            float v = 0.0f;
            for (int r = 0; r < 16; ++r) v += dred[(r * HN + u) * 4 + g];
            a.dbpart[(long)xcd * G4 + g * H + j0 + u] = v;
        }
    }
}

// Launch of 256 workgroups, one per CU.  The kernels need every workgroup of
// an XCD resident at once (consumers wait for producers).  Kernels small
// enough for two workgroups per CU reserve unused LDS so that a CU holds one,
// and on an otherwise idle device a plain dispatch then makes all 256
// resident.  A plain dispatch avoids the queue synchronisation that a
// cooperative launch adds before and after the kernel (about 11 us each).
// Roles are checked in the kernel and every wait has a watchdog, so a launch
// that does not get its workgroups as expected ends every wave and
// lstm_check reports it.  When other kernels may occupy CUs at the same time
// (another stream, collectives overlapping the backward pass),
// LSTM355_XCD_LAUNCH=cooperative selects a cooperative launch, which waits
// until all 256 workgroups can be resident.
constexpr int ONE_PER_CU_LDS = 96 * 1024;   // more than half of a CU's 160 KiB

bool cooperative_requested()
{
    const char *env = std::getenv("LSTM355_XCD_LAUNCH");
    return env && std::strcmp(env, "cooperative") == 0;
}

template <auto kernel>
hipError_t launch256(hipStream_t s, void *argp)
{
    struct Cfg {
        unsigned dyn;
        int per_cu;
    };
    static const Cfg cfg = [] {
        Cfg c{0u, 0};
        hipFuncAttributes fa;
        if (hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(kernel)) != hipSuccess) return c;
        if (fa.sharedSizeBytes < (size_t)ONE_PER_CU_LDS) c.dyn = (unsigned)(ONE_PER_CU_LDS - fa.sharedSizeBytes);
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&c.per_cu, reinterpret_cast<const void *>(kernel), XT,
                                                         c.dyn) != hipSuccess)
            c.per_cu = 0;
        return c;
    }();
    if (cfg.per_cu != 1) return hipErrorCooperativeLaunchTooLarge;
    void *args[] = {argp};
    const void *f = reinterpret_cast<const void *>(kernel);
    if (cooperative_requested())
        return hipLaunchCooperativeKernel(f, dim3(NXCD * WG_PER_XCD), dim3(XT), args, cfg.dyn, s);
    return hipLaunchKernel(f, dim3(NXCD * WG_PER_XCD), dim3(XT), args, cfg.dyn, s);
}

int g_xcd_disabled = 0;

}  // namespace

bool xcd_act16(DType t, const RecShape &sh)
{
    if (t != DType::BF16 || sh.Hp != 0 || (sh.H != 256 && sh.H != 512 && sh.H != 1024)) return false;
    const int RX = (sh.B + NXCD - 1) / NXCD;
    return RX >= 5 && RX <= 32;
}

bool xcd_path_ok(DType t, const RecShape &sh, int num_cus)
{
    if (g_xcd_disabled || t != DType::BF16 || sh.Hp != 0 || num_cus != NXCD * WG_PER_XCD) return false;
    if (sh.H != 256 && sh.H != 512 && sh.H != 1024) return false;
    const int RX = (sh.B + NXCD - 1) / NXCD;
    return RX <= 64;
}

void xcd_path_disable() { g_xcd_disabled = 1; }

namespace {
// FillRanges in one launch: range r is handled by the workgroups with
// blockIdx.y == r, 16-byte stores where the range allows them.
__global__ __launch_bounds__(256) void fill_ranges_kernel(FillRanges f)
{
    const int r = blockIdx.y;
    uint32_t *p = f.p[r];
    const long n = f.n[r];
    const uint32_t v = f.v[r];
    const long stride = (long)gridDim.x * 256;
    const bool vec = (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
    const long nv = vec ? n / 4 : 0;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < nv; i += stride)
        reinterpret_cast<u32x4 *>(p)[i] = u32x4{v, v, v, v};
    for (long i = nv * 4 + (long)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) p[i] = v;
}
}  // namespace

bool wave_path_ok(const RecShape &sh, int num_cus)
{
    return !g_xcd_disabled && num_cus == NXCD * WG_PER_XCD && sh.H == 1024 && sh.Hp == 0 && sh.reverse == 0 &&
           sh.B >= 1 && sh.B <= 32 && sh.ldy == sh.H && (long)sh.T * sh.B * 4L * sh.H * 4 <= 0x7fffffffL;
}

namespace {
// Rows the forward layer wavefront exchanges, armed before its launch: y of
// each layer (dense, two NOT_READY halves per word) and the input projections
// that the projection XCDs write; the flags start at zero.
FillRanges forward_wave_fills(const RecShape &sh, int L, const void *x, const WaveBufs *ly, unsigned *sync)
{
    const long rows = (long)sh.T * sh.B;
    FillRanges f{};
    int nr = 0;
    f.p[nr] = sync + XCD_FLAGS; f.n[nr] = XCD_WORDS; f.v[nr++] = 0u;
    for (int l = 0; l < L && l < 4; ++l) {
        f.p[nr] = static_cast<uint32_t *>(ly[l].y); f.n[nr] = rows * sh.H / 2;
        f.v[nr++] = ((uint32_t)NOT_READY << 16) | NOT_READY;
        if (l > 0 || x) {
            f.p[nr] = reinterpret_cast<uint32_t *>(ly[l].gates); f.n[nr] = rows * 4 * sh.H;
            f.v[nr++] = NOT_READY_F32;
        }
        if (ly[l].sum) {   // residual sums formed in the launch (a layer above may poll them)
            f.p[nr] = static_cast<uint32_t *>(ly[l].sum); f.n[nr] = rows * sh.H / 2;
            f.v[nr++] = ((uint32_t)NOT_READY << 16) | NOT_READY;
        }
    }
    f.count = nr;
    return f;
}
}  // namespace

hipError_t launch_forward_wave(const RecShape &sh, int L, const void *x, const WaveBufs *ly, unsigned *sync,
                               unsigned long long timeout, hipStream_t s)
{
    if (L < 2 || L > 4) return hipErrorInvalidValue;
    XWaveArgs a{};
    a.T = sh.T; a.B = sh.B; a.H = sh.H; a.L = L;
    a.x = static_cast<const bf16_t *>(x);
    bool res = false;
    for (int l = 0; l < L; ++l) {
        a.ly[l].R = static_cast<const bf16_t *>(ly[l].R);
        a.ly[l].W = static_cast<const bf16_t *>(ly[l].W);
        a.ly[l].bias = ly[l].bias;
        a.ly[l].gates = ly[l].gates;
        a.ly[l].cs = ly[l].cs;
        a.ly[l].y = static_cast<bf16_t *>(ly[l].y);
        a.ly[l].in_b = static_cast<const bf16_t *>(ly[l].in_b);
        a.ly[l].sum = static_cast<bf16_t *>(ly[l].sum);
        a.ly[l].poll_b = ly[l].poll_b;
        if (ly[l].in_b) {
            if (l == 0 || !ly[l].sum) return hipErrorInvalidValue;   // a sum is formed from the layer below
            res = true;
        }
    }
    a.flags = sync + XCD_FLAGS;
    a.timeout = timeout;
    const FillRanges f = forward_wave_fills(sh, L, x, ly, sync);
    hipError_t e;
    {
        double bytes = 0.0;
        for (int r = 0; r < f.count; ++r) bytes += 4.0 * f.n[r];
        ProfScope pf(K_SMALL, s, 0.0, bytes);
        hipLaunchKernelGGL(fill_ranges_kernel, dim3(256, f.count), dim3(256), 0, s, f);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    const double G4 = 4.0 * sh.H;
    const int np = x ? L : L - 1;   // input projections computed in the launch
    ProfScope ps(K_REC_FWD, s, 2.0 * sh.T * sh.B * G4 * sh.H * (L + np),
                 (double)L * (sh.T * sh.B * (G4 * 8.0 + sh.H * 6.0) + G4 * sh.H * 2.0) +
                     np * ((double)sh.T * sh.B * (G4 * 4.0 + sh.H * 2.0) + G4 * sh.H * 2.0));
    if (res) {
        if (sh.B <= 16) return launch256<lstm_fwd_wave<32, 1, true>>(s, &a);
        return launch256<lstm_fwd_wave<32, 2, true>>(s, &a);
    }
    if (sh.B <= 16) return launch256<lstm_fwd_wave<32, 1>>(s, &a);
    return launch256<lstm_fwd_wave<32, 2>>(s, &a);
}

FillRanges backward_wave_fills(const RecShape &sh, int L, const WaveBwdBufs *ly, unsigned *sync)
{
    // dz of every layer and the upstream gradients written inside the launch
    // wait for their producers; the flags start at zero
    const long rows = (long)sh.T * sh.B;
    const uint32_t nr2 = ((uint32_t)NOT_READY << 16) | NOT_READY;
    FillRanges f{};
    int nr = 0;
    f.p[nr] = sync + XCD_FLAGS; f.n[nr] = XCD_WORDS; f.v[nr++] = 0u;
    for (int l = 0; l < L && l < 4; ++l) {
        f.p[nr] = static_cast<uint32_t *>(ly[l].dz); f.n[nr] = rows * 4 * sh.H / 2; f.v[nr++] = nr2;
        if (l > 0) { f.p[nr] = static_cast<uint32_t *>(ly[l - 1].dy_fill); f.n[nr] = rows * sh.H / 2; f.v[nr++] = nr2; }
    }
    f.count = nr;
    return f;
}

hipError_t launch_backward_wave(const RecShape &sh, int L, const WaveBwdBufs *ly, unsigned *sync,
                                unsigned long long timeout, hipStream_t s, bool prefilled)
{
    if (L < 2 || L > 4) return hipErrorInvalidValue;
    XWaveBwdArgs a{};
    a.T = sh.T; a.B = sh.B; a.H = sh.H; a.L = L;
    bool res = false;
    for (int l = 0; l < L; ++l) {
        a.ly[l].R = static_cast<const bf16_t *>(ly[l].R);
        a.ly[l].W = static_cast<const bf16_t *>(ly[l].W);
        a.ly[l].gates = ly[l].gates;
        a.ly[l].cs = ly[l].cs;
        a.ly[l].dz = static_cast<bf16_t *>(ly[l].dz);
        a.ly[l].dy = static_cast<const bf16_t *>(ly[l].dy);
        a.ly[l].dx = static_cast<bf16_t *>(ly[l].dx);
        a.ly[l].dbp = ly[l].dbp;
        // a residual layer's input gradient adds its upstream gradient, which
        // the layer above writes in the launch (the stack's own for the top layer)
        if (ly[l].residual) a.res_mask |= 1 << l;
        res = res || (ly[l].residual && ly[l].W);
    }
    a.flags = sync + XCD_FLAGS;
    a.timeout = timeout;
    if (!prefilled) {
        const FillRanges f = backward_wave_fills(sh, L, ly, sync);
        double bytes = 0.0;
        for (int r = 0; r < f.count; ++r) bytes += 4.0 * f.n[r];
        ProfScope pf(K_SMALL, s, 0.0, bytes);
        hipLaunchKernelGGL(fill_ranges_kernel, dim3(256, f.count), dim3(256), 0, s, f);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const double G4 = 4.0 * sh.H;
    int nx = 0;
    for (int l = 0; l < L; ++l) nx += ly[l].W ? 1 : 0;
    ProfScope ps(K_REC_BWD, s, 2.0 * sh.T * sh.B * G4 * sh.H * (L + nx),
                 (double)L * (sh.T * sh.B * (G4 * 4.0 + sh.H * 6.0 + G4 * 2.0) + G4 * sh.H * 2.0) +
                     nx * ((double)sh.T * sh.B * (G4 * 2.0 + sh.H * 2.0) + G4 * sh.H * 2.0));
    if (res) {
        if (sh.B <= 16) return launch256<lstm_bwd_wave<32, 1, true>>(s, &a);
        return launch256<lstm_bwd_wave<32, 2, true>>(s, &a);
    }
    if (sh.B <= 16) return launch256<lstm_bwd_wave<32, 1>>(s, &a);
    return launch256<lstm_bwd_wave<32, 2>>(s, &a);
}

hipError_t xcd_tripped_read_and_clear(unsigned *tripped)
{
    unsigned v = 0;
    hipError_t e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_xcd_tripped), sizeof(v), 0, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return e;
    *tripped = v;
    if (v) {
        const unsigned zero = 0;
        e = hipMemcpyToSymbol(HIP_SYMBOL(g_xcd_tripped), &zero, sizeof(zero), 0, hipMemcpyHostToDevice);
    }
    return e;
}

namespace {
int mbx_for(int B)
{
    const int RX = (B + NXCD - 1) / NXCD;
    const int m = (RX + 15) / 16;
    return m <= 1 ? 1 : (m <= 2 ? 2 : 4);
}
}  // namespace

SideJob xcd_prep_forward(const RecShape &sh, const FwdBufs &bf)
{
    SideJob j;
    j.clr = bf.sync + XCD_FLAGS;
    j.clr_n = XCD_WORDS;
    j.fill = static_cast<uint16_t *>(bf.y);   // the kernel's consumers wait for these elements to change
    j.fill_rows = (long)sh.T * sh.B;
    j.fill_cols = sh.H;
    j.fill_ld = sh.ldy;
    j.fill_v = NOT_READY;
    return j;
}

SideJob xcd_prep_backward(const RecShape &sh, const BwdBufs &bf)
{
    SideJob j;
    j.clr = bf.sync + XCD_FLAGS;
    j.clr_n = XCD_WORDS;
    j.fill = static_cast<uint16_t *>(bf.dz);
    j.fill_rows = (long)sh.T * sh.B;
    j.fill_cols = 4 * sh.H;
    j.fill_ld = 4L * sh.H;
    j.fill_v = NOT_READY;
    return j;
}

hipError_t launch_forward_xcd(const RecShape &sh, const FwdBufs &bf, unsigned long long timeout, hipStream_t s,
                              bool prepared)
{
    XFwdArgs a;
    a.T = sh.T; a.B = sh.B; a.H = sh.H; a.reverse = sh.reverse; a.RX = (sh.B + NXCD - 1) / NXCD; a.ldy = sh.ldy;
    a.R = static_cast<const bf16_t *>(bf.R);
    a.h0 = static_cast<const bf16_t *>(bf.h0);
    a.c0 = bf.c0; a.gates = bf.gates; a.cs = bf.cs;
    a.gx = static_cast<const uint16_t *>(bf.gx16);
    a.act = static_cast<f16_t *>(bf.act16);
    a.y = static_cast<bf16_t *>(bf.y);
    a.hT = static_cast<bf16_t *>(bf.hT);
    a.cT = bf.cT;
    a.flags = bf.sync + XCD_FLAGS;
    a.timeout = timeout;
    if (!prepared) {
        hipError_t e = fill_u32(a.flags, XCD_WORDS, 0u, s);
        if (e != hipSuccess) return e;
        // the kernel's consumers wait for these elements to change
        e = fill_rows_u16(bf.y, (long)sh.T * sh.B, sh.H, sh.ldy, NOT_READY, s);
        if (e != hipSuccess) return e;
    }
    const double G4 = 4.0 * sh.H;
    // per row and step: the input projection read (fp32 or fp16), the
    // activations written (fp32 or fp16), c and h written
    ProfScope ps(K_REC_FWD, s, 2.0 * sh.T * sh.B * G4 * sh.H,
                 (double)sh.T * sh.B * (G4 * ((a.gx ? 2.0 : 4.0) + (a.act ? 2.0 : 4.0)) + sh.H * 6.0) +
                     G4 * sh.H * 2.0);
    const int m = mbx_for(sh.B);
    if ((a.act != nullptr) != xcd_act16(DType::BF16, sh)) return hipErrorInvalidValue;
#define FWD_CASE(HN_, M_)                                                                   \
    if (sh.H == 32 * HN_ && m == M_)                                                        \
        return a.gx ? launch256<lstm_fwd_xcd<HN_, M_, true>>(s, &a) : launch256<lstm_fwd_xcd<HN_, M_>>(s, &a);
#define FWD_CASE_ACT(HN_, M_)                                                                         \
    if (sh.H == 32 * HN_ && m == M_)                                                                  \
        return a.gx ? launch256<lstm_fwd_xcd<HN_, M_, true, true>>(s, &a)                             \
                    : launch256<lstm_fwd_xcd<HN_, M_, false, true>>(s, &a);
    if (a.act) {
        FWD_CASE_ACT(8, 1) FWD_CASE_ACT(8, 2)
        FWD_CASE_ACT(16, 1) FWD_CASE_ACT(16, 2)
        FWD_CASE_ACT(32, 1) FWD_CASE_ACT(32, 2)
        return hipErrorInvalidValue;
    }
    FWD_CASE(8, 1) FWD_CASE(8, 2) FWD_CASE(8, 4)
    FWD_CASE(16, 1) FWD_CASE(16, 2) FWD_CASE(16, 4)
    FWD_CASE(32, 1) FWD_CASE(32, 2) FWD_CASE(32, 4)
#undef FWD_CASE
#undef FWD_CASE_ACT
    return hipErrorInvalidValue;
}

hipError_t launch_backward_xcd(const RecShape &sh, const BwdBufs &bf, unsigned long long timeout, hipStream_t s,
                               bool prepared)
{
    XBwdArgs a;
    a.T = sh.T; a.B = sh.B; a.H = sh.H; a.reverse = sh.reverse; a.RX = (sh.B + NXCD - 1) / NXCD; a.ldy = sh.ldy;
    a.Rt = static_cast<const bf16_t *>(bf.Rt);
    a.dy = static_cast<const bf16_t *>(bf.dy);
    a.dhT = static_cast<const bf16_t *>(bf.dhT);
    a.dcT = bf.dcT; a.c0 = bf.c0; a.gates = bf.gates; a.cs = bf.cs;
    a.act = static_cast<const uint16_t *>(bf.act16);
    a.dz = static_cast<bf16_t *>(bf.dz);
    a.dh0 = static_cast<bf16_t *>(bf.dh0);
    a.dc0 = bf.dc0;
    a.dbpart = bf.dbpart;
    a.flags = bf.sync + XCD_FLAGS;
    a.timeout = timeout;
    if (!prepared) {
        hipError_t e = fill_u32(a.flags, XCD_WORDS, 0u, s);
        if (e != hipSuccess) return e;
        // the kernel's consumers wait for these elements to change
        e = fill_rows_u16(bf.dz, (long)sh.T * sh.B, 4 * sh.H, 4L * sh.H, NOT_READY, s);
        if (e != hipSuccess) return e;
    }
    const double G4 = 4.0 * sh.H;
    // per row and step: the activations (fp32 or fp16), c and dy read, dz written
    ProfScope ps(K_REC_BWD, s, 2.0 * sh.T * sh.B * G4 * sh.H,
                 (double)sh.T * sh.B * (G4 * (a.act ? 2.0 : 4.0) + sh.H * 6.0 + G4 * 2.0) + G4 * sh.H * 2.0);
    const int m = mbx_for(sh.B);
    if ((a.act != nullptr) != xcd_act16(DType::BF16, sh)) return hipErrorInvalidValue;
#define BWD_CASE(HN_, M_) \
    if (sh.H == 32 * HN_ && m == M_) return launch256<lstm_bwd_xcd<HN_, M_>>(s, &a);
#define BWD_CASE_ACT(HN_, M_) \
    if (sh.H == 32 * HN_ && m == M_) return launch256<lstm_bwd_xcd<HN_, M_, true>>(s, &a);
    if (a.act) {
        BWD_CASE_ACT(8, 1) BWD_CASE_ACT(8, 2)
        BWD_CASE_ACT(16, 1) BWD_CASE_ACT(16, 2)
        BWD_CASE_ACT(32, 1) BWD_CASE_ACT(32, 2)
        return hipErrorInvalidValue;
    }
    BWD_CASE(8, 1) BWD_CASE(8, 2) BWD_CASE(8, 4)
    BWD_CASE(16, 1) BWD_CASE(16, 2) BWD_CASE(16, 4)
    BWD_CASE(32, 1) BWD_CASE(32, 2) BWD_CASE(32, 4)
#undef BWD_CASE
#undef BWD_CASE_ACT
    return hipErrorInvalidValue;
}

}  // namespace lstm355
