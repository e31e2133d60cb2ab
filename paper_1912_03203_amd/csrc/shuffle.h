// shuffle.h -- the channel plumbing of a ShuffleNetV2 stride-1 unit whose
// convolutional branch is a gated residual block (Sec. 4.1.2).
//
// The unit splits its C = 2*cb input channels into halves x1 | x2, runs the
// gated block on x2 (Eq. 3) and emits channel_shuffle(concat(x1, b), 2):
// output channel 2k is x1[k], output channel 2k+1 is b[k].  The gated block
// runs on a compact copy of x2 whose rows are zero-extended to cp >= cb
// channels (cp a multiple of 8, what the block kernels take); these two
// kernels move data between the C-channel rows and the cp-channel rows:
//   k_shuffle_split  xa[p] = (x2[p], 0...)                       (first unit)
//   k_shuffle_merge  y[p] = shuffle(x1[p], b[p]); optionally the next unit's
//                    xa[p] = (y[p][cb .. 2cb-1], 0...)
// Both are bandwidth-bound element moves: consecutive threads touch
// consecutive elements of a row, a workgroup a run of whole rows.
#pragma once

#include "kernels.h"

namespace dynconv {

constexpr int kShufRows = 16;  // rows (positions) per workgroup iteration

template <typename T>
__global__ void __launch_bounds__(kBlock)
k_shuffle_split(const T *__restrict__ x, T *__restrict__ xa, int64_t npos, int cb, int cp) {
    const int C = 2 * cb;
    const T zero = static_cast<T>(0.0f);
    for (int64_t p0 = static_cast<int64_t>(blockIdx.x) * kShufRows; p0 < npos;
         p0 += static_cast<int64_t>(gridDim.x) * kShufRows) {
        const int rows = static_cast<int>(npos - p0 < kShufRows ? npos - p0 : kShufRows);
        const T *src = x + p0 * C + cb;
        T *dst = xa + p0 * cp;
        for (int j = threadIdx.x; j < rows * cp; j += kBlock) {
            const int r = j / cp, c = j - r * cp;
            dst[j] = (c < cb) ? src[static_cast<int64_t>(r) * C + c] : zero;
        }
    }
}

template <typename T>
__global__ void __launch_bounds__(kBlock)
k_shuffle_merge(const T *__restrict__ x, const T *__restrict__ br, T *__restrict__ y,
                T *__restrict__ xa, int64_t npos, int cb, int cp) {
    const int C = 2 * cb;
    const T zero = static_cast<T>(0.0f);
    for (int64_t p0 = static_cast<int64_t>(blockIdx.x) * kShufRows; p0 < npos;
         p0 += static_cast<int64_t>(gridDim.x) * kShufRows) {
        const int rows = static_cast<int>(npos - p0 < kShufRows ? npos - p0 : kShufRows);
        const T *xr = x + p0 * C;
        const T *br_r = br + p0 * cp;
        T *yr = y + p0 * C;
        // output channels 2k, 2k+1 of a row: x1[k], b[k]
        for (int j = threadIdx.x; j < rows * cb; j += kBlock) {
            const int r = j / cb, k = j - r * cb;
            T *o = yr + static_cast<int64_t>(r) * C + 2 * k;
            o[0] = xr[static_cast<int64_t>(r) * C + k];
            o[1] = br_r[static_cast<int64_t>(r) * cp + k];
        }
        if (xa) {
            // the next unit's branch input: output channels cb .. 2cb-1
            T *ar = xa + p0 * cp;
            for (int j = threadIdx.x; j < rows * cp; j += kBlock) {
                const int r = j / cp, c = j - r * cp;
                T v = zero;
                if (c < cb) {
                    const int m = cb + c;
                    v = (m & 1) ? br_r[static_cast<int64_t>(r) * cp + (m >> 1)]
                                : xr[static_cast<int64_t>(r) * C + (m >> 1)];
                }
                ar[j] = v;
            }
        }
    }
}

}  // namespace dynconv
