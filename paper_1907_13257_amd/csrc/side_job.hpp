// side_job.hpp -- the device part of SideJob (kernels.hpp): executed by a
// launch's workgroups after their own work.
#pragma once
#include "device_common.hpp"
#include "kernels.hpp"

namespace lstm355 {

// Workgroup `wg` of `nwg` takes its grid-stride share of every part.
__device__ __forceinline__ void run_side_job(const SideJob &j, long wg, long nwg)
{
    const long tid = wg * (long)blockDim.x + threadIdx.x, nth = nwg * (long)blockDim.x;
    if (j.clr)
        for (long i = tid; i < j.clr_n; i += nth) j.clr[i] = 0u;
    if (j.fill && j.fill_ld == j.fill_cols && j.fill_cols % 8 == 0 && (reinterpret_cast<uintptr_t>(j.fill) & 15) == 0) {
        // contiguous rows: one flat range of 16-byte stores, four in flight per thread
        const unsigned v2 = (unsigned)j.fill_v | ((unsigned)j.fill_v << 16);
        const u32x4 v4 = {v2, v2, v2, v2};
        u32x4 *p = reinterpret_cast<u32x4 *>(j.fill);
        const long n = j.fill_rows * j.fill_cols / 8;
        long i = tid;
        for (; i + 3 * nth < n; i += 4 * nth) {
            p[i] = v4;
            p[i + nth] = v4;
            p[i + 2 * nth] = v4;
            p[i + 3 * nth] = v4;
        }
        for (; i < n; i += nth) p[i] = v4;
    } else if (j.fill) {
        const bool vec = j.fill_cols % 8 == 0 && j.fill_ld % 8 == 0 && (reinterpret_cast<uintptr_t>(j.fill) & 15) == 0;
        const long per = vec ? j.fill_cols / 8 : j.fill_cols;
        const long n = j.fill_rows * per;
        const unsigned v2 = (unsigned)j.fill_v | ((unsigned)j.fill_v << 16);
        for (long i = tid; i < n; i += nth) {
            const long r = i / per, c = i % per;
            if (vec)
                *reinterpret_cast<u32x4 *>(j.fill + r * j.fill_ld + c * 8) = u32x4{v2, v2, v2, v2};
            else
                j.fill[r * j.fill_ld + c] = j.fill_v;
        }
    }
    if (j.sum_dst)
        for (long c = tid; c < j.sum_cols; c += nth) {
            float acc = 0.0f;
            for (int r = 0; r < j.sum_rows; ++r) acc += j.sum_src[(long)r * j.sum_cols + c];
            j.sum_dst[c] = j.sum_acc ? j.sum_dst[c] + acc : acc;
        }
}

}  // namespace lstm355
