// dense.h -- the dense layers of a whole MobileNetV2 feature extractor
// (gfx950).  The paper gates only the stride-1 residual blocks; the stem, the
// strided and width-changing blocks and the final 1x1 convolution run on
// every position (Sec. 4.1.2).  All tensors are NHWC, dense, channels
// fastest.
//
//   k_conv1x1    pointwise convolution as a matrix-core contraction:
//                y[p][o] = act(sum_c w[o][c] x[p][c] + b[o]) (+ r[p][o])
//   k_dwconv3x3  depthwise 3x3, stride 1 or 2, zero padding 1, + bias + act
//   k_conv3x3    full 3x3 convolution (the stem: few input channels),
//                stride 1 or 2, zero padding 1, + bias + act
// Output size of the 3x3 layers: (H - 1) / stride + 1.
#pragma once

#include "kernels.h"

namespace dynconv {

// ------------------------------------------------------------ pointwise
// Workgroup tile: 64 positions x 64 outputs, 4 waves; wave w owns positions
// 16w .. 16w+15 of the tile and all 64 outputs (4 MFMA row tiles).  Outputs
// run along M (rows of w), positions along N, so lane (r, g) loads 8
// consecutive channels of one position (B) and of one output row (A) with a
// 16-byte load; the contraction steps through c in 32s, zero past C.
// Every MFMA is issued unconditionally (zero fragments out of range).
constexpr int kPwTile = 64;

template <typename T>
__global__ void __launch_bounds__(kBlock)
k_conv1x1(const T *__restrict__ x, int64_t P, int C, const T *__restrict__ w, const float *__restrict__ b,
          int O, int act, const T *__restrict__ res, T *__restrict__ y) {
    typedef mma<T> M;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const int otiles = (O + kPwTile - 1) / kPwTile;
    const int64_t ptiles = (P + kPwTile - 1) / kPwTile;
    const float lo = act_lo(act), hi = act_hi(act);
    for (int64_t t = blockIdx.x; t < ptiles * otiles; t += gridDim.x) {
        const int64_t pt = t / otiles;
        const int ot = static_cast<int>(t % otiles);
        const int64_t p = pt * kPwTile + wave * 16 + r;  // this lane's position (B column)
        const bool pin = p < P;
        floatx4 acc[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const int o0 = ot * kPwTile + mt * 16 + 4 * g;
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[mt][v] = (o0 + v < O) ? b[o0 + v] : 0.0f;
        }
        for (int c0 = 0; c0 < C; c0 += 32) {
            const int c = c0 + 8 * g;
            const typename M::frag bx = (pin && c < C) ? M::load(x + p * C + c) : M::zero();
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const int o = ot * kPwTile + mt * 16 + r;
                const typename M::frag a =
                    (o < O && c < C) ? M::load(w + static_cast<int64_t>(o) * C + c) : M::zero();
                acc[mt] = M::run(a, bx, acc[mt]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const int o0 = ot * kPwTile + mt * 16 + 4 * g;
            if (pin && o0 < O) {  // O is a multiple of 8: all four outputs exist
                float out[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) out[v] = clamp_act(acc[mt][v], lo, hi);
                if (res) {
                    float rv[4];
                    io<T>::load4(res + p * O + o0, rv);
#pragma unroll
                    for (int v = 0; v < 4; ++v) out[v] += rv[v];
                }
                io<T>::store4(y + p * O + o0, out);
            }
        }
    }
}

// ------------------------------------------------------------ depthwise
// One lane per (output position, 8 channels); the workgroup stages the
// weights transposed, w_t[k][c], and the biases in LDS (dynamic shared
// memory: 9*C elements + C floats).
template <typename T>
__global__ void __launch_bounds__(kBlock)
k_dwconv3x3(const T *__restrict__ x, int N, int H, int W, int C, int stride, const T *__restrict__ w,
            const float *__restrict__ b, int act, T *__restrict__ y, int Ho, int Wo) {
    extern __shared__ __align__(16) unsigned char dw_smem[];
    T *wt = reinterpret_cast<T *>(dw_smem);
    float *bs = reinterpret_cast<float *>(dw_smem + ((9 * C * static_cast<int>(sizeof(T)) + 15) / 16) * 16);
    for (int i = threadIdx.x; i < 9 * C; i += kBlock) {
        const int c = i / 9, k = i % 9;
        wt[k * C + c] = w[i];
    }
    for (int c = threadIdx.x; c < C; c += kBlock) bs[c] = b[c];
    __syncthreads();
    const float lo = act_lo(act), hi = act_hi(act);
    const int groups = C / 8;
    const int64_t total = static_cast<int64_t>(N) * Ho * Wo * groups;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * kBlock) {
        const int c = static_cast<int>(i % groups) * 8;
        const int64_t q = i / groups;  // output position
        const int j = static_cast<int>(q % Wo);
        const int ii = static_cast<int>((q / Wo) % Ho);
        const int n = static_cast<int>(q / (static_cast<int64_t>(Wo) * Ho));
        float s[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) s[u] = bs[c + u];
#pragma unroll
        for (int k = 0; k < 9; ++k) {
            const int hh = stride * ii + k / 3 - 1, ww = stride * j + k % 3 - 1;
            if (hh >= 0 && hh < H && ww >= 0 && ww < W) {
                float v[8], wk[8];
                io<T>::load8(x + ((static_cast<int64_t>(n) * H + hh) * W + ww) * C + c, v);
                io<T>::load8(wt + k * C + c, wk);
#pragma unroll
                for (int u = 0; u < 8; ++u) s[u] = __builtin_fmaf(wk[u], v[u], s[u]);
            }
        }
        float o[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = clamp_act(s[u], lo, hi);
        T *dst = y + q * C + c;
        io<T>::store4(dst, o);
        io<T>::store4(dst + 4, o + 4);
    }
}

// ------------------------------------------------------------ full 3x3
// One lane per (output position, 8 output channels); weights [O][Ci][3][3]
// and biases staged in LDS as fp32, the weights reordered to [k][ci][o] so a
// lane's 8 outputs of one tap and input channel are two 16-byte reads
// (dynamic shared memory: 9*Ci*O + O floats).  Ci is small (the stem's 3
// input channels); input rows are read element by element.
template <typename T>
__global__ void __launch_bounds__(kBlock)
k_conv3x3(const T *__restrict__ x, int N, int H, int W, int Ci, int stride, const T *__restrict__ w,
          const float *__restrict__ b, int O, int act, T *__restrict__ y, int Ho, int Wo) {
    extern __shared__ __align__(16) unsigned char cv_smem[];
    float *ws = reinterpret_cast<float *>(cv_smem);  // [9][Ci][O]
    float *bs = ws + 9 * Ci * O;
    for (int i = threadIdx.x; i < 9 * Ci * O; i += kBlock) {
        const int o = i / (9 * Ci), c = (i / 9) % Ci, k = i % 9;  // w[o][c][k]
        ws[(k * Ci + c) * O + o] = static_cast<float>(w[i]);
    }
    for (int o = threadIdx.x; o < O; o += kBlock) bs[o] = b[o];
    __syncthreads();
    const float lo = act_lo(act), hi = act_hi(act);
    const int groups = O / 8;
    const int64_t total = static_cast<int64_t>(N) * Ho * Wo * groups;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * kBlock) {
        const int o0 = static_cast<int>(i % groups) * 8;
        const int64_t q = i / groups;
        const int j = static_cast<int>(q % Wo);
        const int ii = static_cast<int>((q / Wo) % Ho);
        const int n = static_cast<int>(q / (static_cast<int64_t>(Wo) * Ho));
        float s[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) s[u] = bs[o0 + u];
        for (int k = 0; k < 9; ++k) {
            const int hh = stride * ii + k / 3 - 1, ww = stride * j + k % 3 - 1;
            if (hh < 0 || hh >= H || ww < 0 || ww >= W) continue;
            const T *px = x + ((static_cast<int64_t>(n) * H + hh) * W + ww) * Ci;
            for (int c = 0; c < Ci; ++c) {
                const float v = static_cast<float>(px[c]);
                const float4 wa = *reinterpret_cast<const float4 *>(ws + (k * Ci + c) * O + o0);
                const float4 wb = *reinterpret_cast<const float4 *>(ws + (k * Ci + c) * O + o0 + 4);
                const float wk[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
#pragma unroll
                for (int u = 0; u < 8; ++u) s[u] = __builtin_fmaf(wk[u], v, s[u]);
            }
        }
        float o[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = clamp_act(s[u], lo, hi);
        T *dst = y + q * O + o0;
        io<T>::store4(dst, o);
        io<T>::store4(dst + 4, o + 4);
    }
}

}  // namespace dynconv
