// pointwise.hip -- bandwidth-bound helpers of the LSTM step: weight
// transposes for the backward pass, the bias gradient (column sums of dz),
// stack composition adds, and word fills for barrier counters.
#include "device_common.hpp"
#include "kernels.hpp"

namespace lstm355 {

namespace {

// 64x64 tiles through LDS; both the read and the write are row-contiguous.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T *__restrict__ src, int rows, int cols, T *__restrict__ dst)
{
    __shared__ T tile[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4)
        if (r0 + i < rows && c0 + tx < cols) tile[i][tx] = src[(long)(r0 + i) * cols + c0 + tx];
    __syncthreads();
    for (int i = ty; i < 64; i += 4)
        if (c0 + i < cols && r0 + tx < rows) dst[(long)(c0 + i) * rows + r0 + tx] = tile[tx][i];
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

constexpr int CS_ROWS = 256;   // rows per partial sum

// Pass 1: partial[chunk][c] = sum of rows [chunk*256, chunk*256+256) of column c.
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

int grid_for(size_t n)
{
    size_t g = (n + 255) / 256;
    if (g > 8192) g = 8192;
    return g ? (int)g : 1;
}

}  // namespace

hipError_t transpose(DType t, const void *src, int rows, int cols, void *dst, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, 2.0 * rows * (double)cols * dsize(t));
    dim3 grid((cols + 63) / 64, (rows + 63) / 64);
    if (t == DType::BF16)
        hipLaunchKernelGGL(transpose_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<const bf16_t *>(src), rows,
                           cols, static_cast<bf16_t *>(dst));
    else
        hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, static_cast<const float *>(src), rows, cols,
                           static_cast<float *>(dst));
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

hipError_t add(DType t, size_t n, const void *a, const void *b, void *out, hipStream_t s)
{
    ProfScope ps(K_SMALL, s, 0.0, 3.0 * n * dsize(t));
    if (t == DType::BF16)
        hipLaunchKernelGGL(add_kernel<bf16_t>, dim3(grid_for(n)), dim3(256), 0, s, n, static_cast<const bf16_t *>(a),
                           static_cast<const bf16_t *>(b), static_cast<bf16_t *>(out));
    else
        hipLaunchKernelGGL(add_kernel<float>, dim3(grid_for(n)), dim3(256), 0, s, n, static_cast<const float *>(a),
                           static_cast<const float *>(b), static_cast<float *>(out));
    return hipGetLastError();
}

}  // namespace lstm355
