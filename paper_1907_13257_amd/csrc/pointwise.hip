// pointwise.hip -- bandwidth-bound helpers of the LSTM step: weight
// transposes for the backward pass, the bias gradient (column sums of dz),
// stack composition adds, and word fills for barrier counters.
#include "device_common.hpp"
#include "kernels.hpp"
#include "side_job.hpp"

namespace lstm355 {

namespace {

// 64x64 tiles through LDS; both the read and the write are row-contiguous.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T *__restrict__ src, int rows, int cols, T *__restrict__ dst,
                                                        SideJob side)
{
    __shared__ T tile[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4)
        if (r0 + i < rows && c0 + tx < cols) tile[i][tx] = src[(long)(r0 + i) * cols + c0 + tx];
    __syncthreads();
    for (int i = ty; i < 64; i += 4)
        if (c0 + i < cols && r0 + tx < rows) dst[(long)(c0 + i) * rows + r0 + tx] = tile[tx][i];
    run_side_job(side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
}

// 16-bit elements, rows and cols multiples of 64, 16-byte aligned: 16-byte
// loads along the source rows and 16-byte stores along the destination rows.
__device__ __forceinline__ void transpose_u16_vec_tile(const uint16_t *__restrict__ src, int rows, int cols,
                                                       uint16_t *__restrict__ dst)
{
    __shared__ uint16_t tile[64][72];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int t = threadIdx.x, q = t & 7;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const int i = p * 32 + (t >> 3);
        const u32x4 v = *reinterpret_cast<const u32x4 *>(src + (long)(r0 + i) * cols + c0 + q * 8);
        *reinterpret_cast<u32x4 *>(&tile[i][q * 8]) = v;
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const int i = p * 32 + (t >> 3);   // destination row c0 + i, source rows r0 + q*8 .. +8
        unsigned w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
            w[e] = (unsigned)tile[q * 8 + 2 * e][i] | ((unsigned)tile[q * 8 + 2 * e + 1][i] << 16);
        *reinterpret_cast<u32x4 *>(dst + (long)(c0 + i) * rows + r0 + q * 8) = u32x4{w[0], w[1], w[2], w[3]};
    }
}

__global__ __launch_bounds__(256) void transpose_u16_vec_kernel(const uint16_t *__restrict__ src, int rows, int cols,
                                                                uint16_t *__restrict__ dst, SideJob side)
{
    transpose_u16_vec_tile(src, rows, cols, dst);
    run_side_job(side, (long)blockIdx.y * gridDim.x + blockIdx.x, (long)gridDim.x * gridDim.y);
}

__global__ void fill_kernel(uint32_t *p, size_t n, uint32_t v)
{
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// 16-bit fill of a strided row range; 16-byte stores when rows are 8-element aligned.
__global__ void fill_rows_u16_kernel(uint16_t *p, long rows, int cols, long ld, uint16_t v, int vec)
{
    const long per_row = vec ? cols / 8 : cols;
    const long n = rows * per_row;
    const unsigned v2 = (unsigned)v | ((unsigned)v << 16);
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        const long r = i / per_row, c = i % per_row;
        if (vec)
            *reinterpret_cast<u32x4 *>(p + r * ld + c * 8) = u32x4{v2, v2, v2, v2};
        else
            p[r * ld + c] = v;
    }
}

constexpr int CS_ROWS = 64;   // rows per partial sum

// Pass 1: partial[chunk][c] = sum of rows [chunk*CS_ROWS, (chunk+1)*CS_ROWS) of column c.
template <typename T>
__global__ __launch_bounds__(256) void colsum_pass1(const T *__restrict__ src, int rows, int cols, float *__restrict__ partial)
{
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int chunk = blockIdx.y;
    if (c >= cols) return;
    const int r1 = min(rows, (chunk + 1) * CS_ROWS);
    float acc = 0.0f;
    for (int r = chunk * CS_ROWS; r < r1; ++r) acc += to_f32(src[(long)r * cols + c]);
    partial[(long)chunk * cols + c] = acc;
}

// The same with 16-byte loads: each thread sums E = 16 / sizeof(T) adjacent
// columns (cols a multiple of E, src 16-byte aligned), eight rows in flight.
template <typename T>
__global__ __launch_bounds__(256) void colsum_pass1_vec(const T *__restrict__ src, int rows, int cols,
                                                        float *__restrict__ partial)
{
    constexpr int E = 16 / (int)sizeof(T);
    const int c = (blockIdx.x * 256 + threadIdx.x) * E;
    const int chunk = blockIdx.y;
    if (c >= cols) return;
    const int r0 = chunk * CS_ROWS, r1 = min(rows, r0 + CS_ROWS);
    float acc[E];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.0f;
    const char *base = reinterpret_cast<const char *>(src + c);
    const long pitch = (long)cols * (long)sizeof(T);
#pragma unroll 8
    for (int r = r0; r < r1; ++r) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(base + (long)r * pitch);
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc[2 * q] += __uint_as_float(v[q] << 16);
                acc[2 * q + 1] += __uint_as_float(v[q] & 0xffff0000u);
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] += __uint_as_float(v[q]);
        }
    }
    float *out = partial + (long)chunk * cols + c;
#pragma unroll
    for (int e = 0; e < E; e += 4) *reinterpret_cast<f32x4 *>(out + e) = f32x4{acc[e], acc[e + 1], acc[e + 2], acc[e + 3]};
}

// Pass 2: dst[c] (+)= sum over chunks, in chunk order.
__global__ __launch_bounds__(256) void colsum_pass2(const float *__restrict__ partial, int nchunk, int cols, float *dst, int accumulate)
{
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= cols) return;
    float acc = 0.0f;
    for (int k = 0; k < nchunk; ++k) acc += partial[(long)k * cols + c];
    dst[c] = accumulate ? dst[c] + acc : acc;
}

template <typename T>
__global__ __launch_bounds__(256) void add_kernel(size_t n, const T *a, const T *b, T *out)
{
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        out[i] = from_f32<T>(to_f32(a[i]) + to_f32(b[i]));
}

// The same with 16-byte accesses (n a multiple of 16 / sizeof(T), all three
// pointers 16-byte aligned); per element the same arithmetic and rounding.
template <typename T>
__global__ __launch_bounds__(256) void add_kernel_vec(size_t nv, const T *a, const T *b, T *out)
{
    constexpr int E = 16 / (int)sizeof(T);
    const u32x4 *av = reinterpret_cast<const u32x4 *>(a), *bv = reinterpret_cast<const u32x4 *>(b);
    u32x4 *ov = reinterpret_cast<u32x4 *>(out);
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += (size_t)gridDim.x * blockDim.x) {
        const u32x4 x = av[i], y = bv[i];
        T xs[E], ys[E], r[E];
        __builtin_memcpy(xs, &x, 16);
        __builtin_memcpy(ys, &y, 16);
#pragma unroll
        for (int e = 0; e < E; ++e) r[e] = from_f32<T>(to_f32(xs[e]) + to_f32(ys[e]));
        u32x4 o;
        __builtin_memcpy(&o, r, 16);
        ov[i] = o;
    }
}

// One step of the cell update for every (row b, cell j), after the
// recurrent product has been added to the step's input projection:
// z = gates_t (pre-activations in, activations i, f, g, o out, in place);
// c_t = f c_{t-1} + i g; m_t = o tanh(c_t).
template <typename TI>
__global__ __launch_bounds__(256) void gates_forward_kernel(int B, int H, float *__restrict__ gates,
                                                            const float *__restrict__ cprev, float *__restrict__ c_t,
                                                            TI *__restrict__ m_out, long ldm, TI *__restrict__ h_copy,
                                                            long ldh, float *__restrict__ cT)
{
    const long n = (long)B * H;
    for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
        const int b = (int)(e / H), j = (int)(e % H);
        float *g = gates + (long)b * 4 * H + j;
        const float ig = sigmoid_f(g[0]), fg = sigmoid_f(g[H]), gg = tanh_f(g[2 * H]), og = sigmoid_f(g[3 * H]);
        const float cp = cprev ? cprev[e] : 0.0f;
        const float c = fg * cp + ig * gg;
        const TI m = from_f32<TI>(og * tanh_f(c));
        g[0] = ig;
        g[H] = fg;
        g[2 * H] = gg;
        g[3 * H] = og;
        c_t[e] = c;
        m_out[(long)b * ldm + j] = m;
        if (h_copy) h_copy[(long)b * ldh + j] = m;
        if (cT) cT[e] = c;
    }
}

// Gate gradients of one step for every (row b, cell j).  The gradient of
// m_t is the sum of the given terms: dm (fp32), dy (storage type, row
// stride ldy), dh (fp32) and dhT (storage type).  dcn carries the cell
// gradient between steps (in: from step t+1, out: to step t-1).
template <typename TI>
__global__ __launch_bounds__(256) void gates_backward_kernel(int B, int H, const float *__restrict__ dm_in,
                                                             const TI *__restrict__ dy, long ldy,
                                                             const float *__restrict__ dh_in, const TI *__restrict__ dhT,
                                                             const float *__restrict__ gates, const float *__restrict__ c_t,
                                                             const float *__restrict__ cprev, float *__restrict__ dcn,
                                                             TI *__restrict__ dz, float *__restrict__ dc0)
{
    const long n = (long)B * H;
    for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
        const int b = (int)(e / H), j = (int)(e % H);
        float dm = 0.0f;
        if (dm_in) dm += dm_in[e];
        if (dy) dm += to_f32(dy[(long)b * ldy + j]);
        if (dh_in) dm += dh_in[e];
        if (dhT) dm += to_f32(dhT[e]);
        const float *g = gates + (long)b * 4 * H + j;
        const float ig = g[0], fg = g[H], gg = g[2 * H], og = g[3 * H];
        const float tc = tanh_f(c_t[e]);
        const float d_o = dm * tc;
        const float d_c = dcn[e] + dm * og * (1.0f - tc * tc);
        const float cp = cprev ? cprev[e] : 0.0f;
        const float d_i = d_c * gg, d_g = d_c * ig, d_f = d_c * cp;
        TI *z = dz + (long)b * 4 * H + j;
        z[0] = from_f32<TI>(d_i * ig * (1.0f - ig));
        z[H] = from_f32<TI>(d_f * fg * (1.0f - fg));
        z[2 * H] = from_f32<TI>(d_g * (1.0f - gg * gg));
        z[3 * H] = from_f32<TI>(d_o * og * (1.0f - og));
        const float nc = d_c * fg;
        dcn[e] = nc;
        if (dc0) dc0[e] = nc;
    }
}

// The same for four adjacent cells per thread (H a multiple of 4, ldy a
// multiple of 4, every pointer 16-byte aligned): 16-byte fp32 and 8-byte
// bf16 accesses, the same arithmetic per cell.
__device__ __forceinline__ f32x4 ld4(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }
__device__ __forceinline__ void ld4(const bf16_t *p, float (&o)[4])
{
    const u32x2 v = *reinterpret_cast<const u32x2 *>(p);
    o[0] = __uint_as_float(v[0] << 16);
    o[1] = __uint_as_float(v[0] & 0xffff0000u);
    o[2] = __uint_as_float(v[1] << 16);
    o[3] = __uint_as_float(v[1] & 0xffff0000u);
}
__device__ __forceinline__ void ld4(const float *p, float (&o)[4])
{
    const f32x4 v = ld4(p);
    o[0] = v[0]; o[1] = v[1]; o[2] = v[2]; o[3] = v[3];
}
__device__ __forceinline__ void st4(bf16_t *p, const float (&v)[4])
{
    const unsigned lo = (unsigned)f32_to_bf16(v[0]) | ((unsigned)f32_to_bf16(v[1]) << 16);
    const unsigned hi = (unsigned)f32_to_bf16(v[2]) | ((unsigned)f32_to_bf16(v[3]) << 16);
    *reinterpret_cast<u32x2 *>(p) = u32x2{lo, hi};
}
__device__ __forceinline__ void st4(float *p, const float (&v)[4])
{
    *reinterpret_cast<f32x4 *>(p) = f32x4{v[0], v[1], v[2], v[3]};
}

template <typename TI>
__global__ __launch_bounds__(256) void gates_backward4_kernel(int B, int H, const float *__restrict__ dm_in,
                                                              const TI *__restrict__ dy, long ldy,
                                                              const float *__restrict__ dh_in, const TI *__restrict__ dhT,
                                                              const float *__restrict__ gates,
                                                              const float *__restrict__ c_t,
                                                              const float *__restrict__ cprev, float *__restrict__ dcn,
                                                              TI *__restrict__ dz, float *__restrict__ dc0)
{
    const long n4 = (long)B * H / 4;
    for (long q = (long)blockIdx.x * blockDim.x + threadIdx.x; q < n4; q += (long)gridDim.x * blockDim.x) {
        const long e = q * 4;
        const int b = (int)(e / H), j = (int)(e % H);
        float dm[4] = {0.f, 0.f, 0.f, 0.f}, t4[4];
        if (dm_in) { ld4(dm_in + e, t4); for (int k = 0; k < 4; ++k) dm[k] += t4[k]; }
        if (dy) { ld4(dy + (long)b * ldy + j, t4); for (int k = 0; k < 4; ++k) dm[k] += t4[k]; }
        if (dh_in) { ld4(dh_in + e, t4); for (int k = 0; k < 4; ++k) dm[k] += t4[k]; }
        if (dhT) { ld4(dhT + e, t4); for (int k = 0; k < 4; ++k) dm[k] += t4[k]; }
        const float *g = gates + (long)b * 4 * H + j;
        const f32x4 ig = ld4(g), fg = ld4(g + H), gg = ld4(g + 2 * H), og = ld4(g + 3 * H);
        const f32x4 c4 = ld4(c_t + e), dcn4 = ld4(dcn + e);
        const f32x4 cp4 = cprev ? ld4(cprev + e) : f32x4{0.f, 0.f, 0.f, 0.f};
        float zi[4], zf[4], zg[4], zo[4], nc[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float tc = tanh_f(c4[k]);
            const float d_o = dm[k] * tc;
            const float d_c = dcn4[k] + dm[k] * og[k] * (1.0f - tc * tc);
            const float d_i = d_c * gg[k], d_g = d_c * ig[k], d_f = d_c * cp4[k];
            zi[k] = d_i * ig[k] * (1.0f - ig[k]);
            zf[k] = d_f * fg[k] * (1.0f - fg[k]);
            zg[k] = d_g * (1.0f - gg[k] * gg[k]);
            zo[k] = d_o * og[k] * (1.0f - og[k]);
            nc[k] = d_c * fg[k];
        }
        TI *z = dz + (long)b * 4 * H + j;
        st4(z, zi);
        st4(z + H, zf);
        st4(z + 2 * H, zg);
        st4(z + 3 * H, zo);
        st4(dcn + e, nc);
        if (dc0) st4(dc0 + e, nc);
    }
}

template <typename T>
__global__ __launch_bounds__(256) void copy_rows_kernel(long rows, int cols, const T *__restrict__ src, long lds,
                                                        T *__restrict__ dst, long ldd)
{
    const long n = rows * cols;
    for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
        const long r = e / cols, c = e % cols;
        dst[r * ldd + c] = src[r * lds + c];
    }
}

int grid_for(size_t n)
{
    size_t g = (n + 255) / 256;
    if (g > 8192) g = 8192;
    return g ? (int)g : 1;
}

}  // namespace

hipError_t transpose(DType t, const void *src, int rows, int cols, void *dst, hipStream_t s, const SideJob *side)
{
    ProfScope ps(K_SMALL, s, 0.0, 2.0 * rows * (double)cols * dsize(t));
    dim3 grid((cols + 63) / 64, (rows + 63) / 64);
    const SideJob sj = side ? *side : SideJob{};
    if (t == DType::BF16 && rows % 64 == 0 && cols % 64 == 0 &&
        ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15) == 0) {
        hipLaunchKernelGGL(transpose_u16_vec_kernel, grid, dim3(256), 0, s, static_cast<const uint16_t *>(src), rows,
                           cols, static_cast<uint16_t *>(dst), sj);
        return hipGetLastError();
    }
    if (t == DType::BF16)
        hipLaunchKernelGGL(transpose_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<const bf16_t *>(src), rows,
                           cols, static_cast<bf16_t *>(dst), sj);
    else
        hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, static_cast<const float *>(src), rows, cols,
                           static_cast<float *>(dst), sj);
    return hipGetLastError();
}

hipError_t fill_u32(void *p, size_t n, uint32_t v, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, 4.0 * n);
    hipLaunchKernelGGL(fill_kernel, dim3(grid_for(n)), dim3(256), 0, s, static_cast<uint32_t *>(p), n, v);
    return hipGetLastError();
}

hipError_t fill_rows_u16(void *p, long rows, int cols, long ld, uint16_t v, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, 2.0 * rows * cols);
    const int vec = (cols % 8 == 0 && ld % 8 == 0 && (reinterpret_cast<uintptr_t>(p) & 15) == 0) ? 1 : 0;
    const size_t n = (size_t)rows * (vec ? cols / 8 : cols);
    hipLaunchKernelGGL(fill_rows_u16_kernel, dim3(grid_for(n)), dim3(256), 0, s, static_cast<uint16_t *>(p), rows, cols,
                       ld, v, vec);
    return hipGetLastError();
}

size_t colsum_partial_floats(int rows, int cols) { return (size_t)((rows + CS_ROWS - 1) / CS_ROWS) * cols; }

hipError_t colsum(DType t, const void *src, int rows, int cols, float *partial, float *dst, int accumulate, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, (double)rows * cols * dsize(t));
    const int nchunk = (rows + CS_ROWS - 1) / CS_ROWS;
    const int E = 16 / (int)dsize(t);
    if (cols % E == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0 && (reinterpret_cast<uintptr_t>(partial) & 15) == 0) {
        dim3 gv((cols / E + 255) / 256, nchunk);
        if (t == DType::BF16)
            hipLaunchKernelGGL(colsum_pass1_vec<bf16_t>, gv, dim3(256), 0, s, static_cast<const bf16_t *>(src), rows, cols,
                               partial);
        else
            hipLaunchKernelGGL(colsum_pass1_vec<float>, gv, dim3(256), 0, s, static_cast<const float *>(src), rows, cols,
                               partial);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(colsum_pass2, dim3((cols + 255) / 256), dim3(256), 0, s, partial, nchunk, cols, dst, accumulate);
        return hipGetLastError();
    }
    dim3 g1((cols + 255) / 256, nchunk);
    if (t == DType::BF16)
        hipLaunchKernelGGL(colsum_pass1<bf16_t>, g1, dim3(256), 0, s, static_cast<const bf16_t *>(src), rows, cols, partial);
    else
        hipLaunchKernelGGL(colsum_pass1<float>, g1, dim3(256), 0, s, static_cast<const float *>(src), rows, cols, partial);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(colsum_pass2, dim3((cols + 255) / 256), dim3(256), 0, s, partial, nchunk, cols, dst, accumulate);
    return hipGetLastError();
}

hipError_t sum_rows(const float *src, int rows, int cols, float *dst, int accumulate, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, (double)rows * cols * 4.0);
    hipLaunchKernelGGL(colsum_pass2, dim3((cols + 255) / 256), dim3(256), 0, s, src, rows, cols, dst, accumulate);
    return hipGetLastError();
}

hipError_t gates_forward(DType t, int B, int H, float *gates_t, const float *cprev, float *c_t, void *m_out, long ldm,
                         void *h_copy, long ldh, float *cT, int kclass, hipStream_t s)
{
    const double n = (double)B * H;
    ProfScope ps(kclass, s, 0.0, n * (4.0 * 4 * 2 + 4.0 * (cprev ? 2 : 1) + dsize(t) * (h_copy ? 2 : 1)));
    const size_t ne = (size_t)B * H;
    if (t == DType::BF16)
        hipLaunchKernelGGL(gates_forward_kernel<bf16_t>, dim3(grid_for(ne)), dim3(256), 0, s, B, H, gates_t, cprev, c_t,
                           static_cast<bf16_t *>(m_out), ldm, static_cast<bf16_t *>(h_copy), ldh, cT);
    else
        hipLaunchKernelGGL(gates_forward_kernel<float>, dim3(grid_for(ne)), dim3(256), 0, s, B, H, gates_t, cprev, c_t,
                           static_cast<float *>(m_out), ldm, static_cast<float *>(h_copy), ldh, cT);
    return hipGetLastError();
}

hipError_t gates_backward(DType t, int B, int H, const float *dm, const void *dy, long ldy, const float *dh,
                          const void *dhT, const float *gates_t, const float *c_t, const float *cprev, float *dcn,
                          void *dz_t, float *dc0, int kclass, hipStream_t s)
{
    const double n = (double)B * H;
    ProfScope ps(kclass, s, 0.0, n * (4.0 * 4 + 4.0 * 4 + dsize(t) * 4));
    const size_t ne = (size_t)B * H;
    const uintptr_t al = reinterpret_cast<uintptr_t>(dm) | reinterpret_cast<uintptr_t>(dy) |
                         reinterpret_cast<uintptr_t>(dh) | reinterpret_cast<uintptr_t>(dhT) |
                         reinterpret_cast<uintptr_t>(gates_t) | reinterpret_cast<uintptr_t>(c_t) |
                         reinterpret_cast<uintptr_t>(cprev) | reinterpret_cast<uintptr_t>(dcn) |
                         reinterpret_cast<uintptr_t>(dz_t) | reinterpret_cast<uintptr_t>(dc0);
    if (H % 4 == 0 && ldy % 4 == 0 && (al & 15) == 0) {
        if (t == DType::BF16)
            hipLaunchKernelGGL(gates_backward4_kernel<bf16_t>, dim3(grid_for(ne / 4)), dim3(256), 0, s, B, H, dm,
                               static_cast<const bf16_t *>(dy), ldy, dh, static_cast<const bf16_t *>(dhT), gates_t, c_t,
                               cprev, dcn, static_cast<bf16_t *>(dz_t), dc0);
        else
            hipLaunchKernelGGL(gates_backward4_kernel<float>, dim3(grid_for(ne / 4)), dim3(256), 0, s, B, H, dm,
                               static_cast<const float *>(dy), ldy, dh, static_cast<const float *>(dhT), gates_t, c_t,
                               cprev, dcn, static_cast<float *>(dz_t), dc0);
        return hipGetLastError();
    }
    if (t == DType::BF16)
        hipLaunchKernelGGL(gates_backward_kernel<bf16_t>, dim3(grid_for(ne)), dim3(256), 0, s, B, H, dm,
                           static_cast<const bf16_t *>(dy), ldy, dh, static_cast<const bf16_t *>(dhT), gates_t, c_t,
                           cprev, dcn, static_cast<bf16_t *>(dz_t), dc0);
    else
        hipLaunchKernelGGL(gates_backward_kernel<float>, dim3(grid_for(ne)), dim3(256), 0, s, B, H, dm,
                           static_cast<const float *>(dy), ldy, dh, static_cast<const float *>(dhT), gates_t, c_t,
                           cprev, dcn, static_cast<float *>(dz_t), dc0);
    return hipGetLastError();
}

hipError_t copy_rows(DType t, long rows, int cols, const void *src, long lds, void *dst, long ldd, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, 2.0 * rows * cols * dsize(t));
    const size_t ne = (size_t)rows * cols;
    if (t == DType::BF16)
        hipLaunchKernelGGL(copy_rows_kernel<bf16_t>, dim3(grid_for(ne)), dim3(256), 0, s, rows, cols,
                           static_cast<const bf16_t *>(src), lds, static_cast<bf16_t *>(dst), ldd);
    else
        hipLaunchKernelGGL(copy_rows_kernel<float>, dim3(grid_for(ne)), dim3(256), 0, s, rows, cols,
                           static_cast<const float *>(src), lds, static_cast<float *>(dst), ldd);
    return hipGetLastError();
}

hipError_t add(DType t, size_t n, const void *a, const void *b, void *out, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, 3.0 * n * dsize(t));
    const size_t E = 16 / dsize(t);
    const uintptr_t align = reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) | reinterpret_cast<uintptr_t>(out);
    if (n % E == 0 && (align & 15) == 0) {
        const size_t nv = n / E;
        if (t == DType::BF16)
            hipLaunchKernelGGL(add_kernel_vec<bf16_t>, dim3(grid_for(nv)), dim3(256), 0, s, nv,
                               static_cast<const bf16_t *>(a), static_cast<const bf16_t *>(b), static_cast<bf16_t *>(out));
        else
            hipLaunchKernelGGL(add_kernel_vec<float>, dim3(grid_for(nv)), dim3(256), 0, s, nv,
                               static_cast<const float *>(a), static_cast<const float *>(b), static_cast<float *>(out));
        return hipGetLastError();
    }
    if (t == DType::BF16)
        hipLaunchKernelGGL(add_kernel<bf16_t>, dim3(grid_for(n)), dim3(256), 0, s, n, static_cast<const bf16_t *>(a),
                           static_cast<const bf16_t *>(b), static_cast<bf16_t *>(out));
    else
        hipLaunchKernelGGL(add_kernel<float>, dim3(grid_for(n)), dim3(256), 0, s, n, static_cast<const float *>(a),
                           static_cast<const float *>(b), static_cast<float *>(out));
    return hipGetLastError();
}

}  // namespace lstm355
