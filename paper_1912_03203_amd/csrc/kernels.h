// kernels.h -- gfx950 (CDNA4) device code for the spatially gated
// inverted-residual block of Verelst & Tuytelaars (CVPR 2020), Sec. 3.2.
//
// Kernel chain for one gated block (one stream, no host synchronisation):
//   k_mask        mask unit + hard threshold (Eq. 2, Eq. 8 at zero noise)
//   k_rowcount    per image row: active and dilated counts
//   k_rowscan     exclusive scan of the row counts -> row offsets, P, P_d
//   k_compact     per image row: ballot ranks -> active / dilated lists and
//                 the neighbour table of the modified depthwise convolution
//   k_expand      gather of the dilated rows + 1x1 expansion on the matrix
//                 cores (fp32 accumulation) + bias + activation
//   k_dw_project  depthwise 3x3 at the active rows through the neighbour
//                 table, 1x1 projection on the matrix cores, bias, and the
//                 scatter-add into the identity path
// The dense baseline (Eq. 1) runs k_expand and k_dw_project with identity
// addressing over every position.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dynconv {

typedef _Float16 half_t;
typedef __bf16 bf16_t;
typedef half_t half8 __attribute__((ext_vector_type(8)));
typedef half_t half4 __attribute__((ext_vector_type(4)));
typedef bf16_t bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16_t bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;          // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kMaxSeg = 64;          // image width limit: 64 segments of 64 columns

// ---------------------------------------------------------------- storage I/O
// load8: 8 consecutive elements -> fp32 (exact widening).
// store4: 4 fp32 values -> 4 consecutive elements (round to nearest even).
template <typename T> struct io;

template <> struct io<float> {
    struct vec8 {
        float v[8];
        __device__ __forceinline__ float operator[](int i) const { return v[i]; }
    };
    static __device__ __forceinline__ vec8 raw8(const float *p) {
        vec8 r;
        load8(p, r.v);
        return r;
    }
    static __device__ __forceinline__ void load8(const float *p, float v[8]) {
        float4 a = *reinterpret_cast<const float4 *>(p);
        float4 b = *reinterpret_cast<const float4 *>(p + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
    static __device__ __forceinline__ void load4(const float *p, float v[4]) {
        float4 a = *reinterpret_cast<const float4 *>(p);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    }
    static __device__ __forceinline__ void store4(float *p, const float v[4]) {
        *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
    }
};

template <> struct io<half_t> {
    typedef half8 vec8;  // 8 values packed in 4 registers
    static __device__ __forceinline__ vec8 raw8(const half_t *p) {
        return *reinterpret_cast<const half8 *>(p);
    }
    static __device__ __forceinline__ void load8(const half_t *p, float v[8]) {
        half8 h = *reinterpret_cast<const half8 *>(p);
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = static_cast<float>(h[u]);
    }
    static __device__ __forceinline__ void load4(const half_t *p, float v[4]) {
        half4 h = *reinterpret_cast<const half4 *>(p);
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = static_cast<float>(h[u]);
    }
    static __device__ __forceinline__ void store4(half_t *p, const float v[4]) {
        half4 h;
#pragma unroll
        for (int u = 0; u < 4; ++u) h[u] = static_cast<half_t>(v[u]);
        *reinterpret_cast<half4 *>(p) = h;
    }
};

template <> struct io<bf16_t> {
    typedef bf16x8 vec8;
    static __device__ __forceinline__ vec8 raw8(const bf16_t *p) {
        return *reinterpret_cast<const bf16x8 *>(p);
    }
    static __device__ __forceinline__ void load8(const bf16_t *p, float v[8]) {
        bf16x8 h = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = static_cast<float>(h[u]);
    }
    static __device__ __forceinline__ void load4(const bf16_t *p, float v[4]) {
        bf16x4 h = *reinterpret_cast<const bf16x4 *>(p);
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = static_cast<float>(h[u]);
    }
    static __device__ __forceinline__ void store4(bf16_t *p, const float v[4]) {
        bf16x4 h;
#pragma unroll
        for (int u = 0; u < 4; ++u) h[u] = static_cast<bf16_t>(v[u]);
        *reinterpret_cast<bf16x4 *>(p) = h;
    }
};

// ------------------------------------------------------------ matrix cores
// One 16x16 output tile per wave.  Lane l = 16*g + r (r = l % 16, g = l / 16)
// supplies row r of the A tile and column r of the B tile, each as 8
// consecutive entries of a 32-long slice of the contraction dimension starting
// at 8*g; A and B use the same slice assignment, so the product sums over the
// full slice.  The accumulator lane l holds D[4*g + v][r], v = 0..3.
// fp16/bf16: one v_mfma_f32_16x16x32_{f16,bf16}; fp32: eight
// v_mfma_f32_16x16x4_f32, the j-th one pairing entry j of every lane.
template <typename T> struct mma;

template <> struct mma<half_t> {
    typedef half8 frag;
    static __device__ __forceinline__ frag zero() { return frag{}; }
    static __device__ __forceinline__ frag load(const half_t *p) {
        return *reinterpret_cast<const half8 *>(p);
    }
    static __device__ __forceinline__ frag pack(const float v[8]) {
        frag f;
#pragma unroll
        for (int u = 0; u < 8; ++u) f[u] = static_cast<half_t>(v[u]);
        return f;
    }
    static __device__ __forceinline__ floatx4 run(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};

template <> struct mma<bf16_t> {
    typedef bf16x8 frag;
    static __device__ __forceinline__ frag zero() { return frag{}; }
    static __device__ __forceinline__ frag load(const bf16_t *p) {
        return *reinterpret_cast<const bf16x8 *>(p);
    }
    static __device__ __forceinline__ frag pack(const float v[8]) {
        frag f;
#pragma unroll
        for (int u = 0; u < 8; ++u) f[u] = static_cast<bf16_t>(v[u]);
        return f;
    }
    static __device__ __forceinline__ floatx4 run(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

struct f32frag {
    float v[8];
};

template <> struct mma<float> {
    typedef f32frag frag;
    static __device__ __forceinline__ frag zero() {
        frag f;
#pragma unroll
        for (int u = 0; u < 8; ++u) f.v[u] = 0.0f;
        return f;
    }
    static __device__ __forceinline__ frag load(const float *p) {
        frag f;
        io<float>::load8(p, f.v);
        return f;
    }
    static __device__ __forceinline__ frag pack(const float v[8]) {
        frag f;
#pragma unroll
        for (int u = 0; u < 8; ++u) f.v[u] = v[u];
        return f;
    }
    static __device__ __forceinline__ floatx4 run(frag a, frag b, floatx4 c) {
#pragma unroll
        for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], c, 0, 0, 0);
        return c;
    }
};

// Activation as one clamp: kind 0 none, 1 ReLU, 2 ReLU6.  act_lo / act_hi
// are uniform, so activate() is a single branch-free v_med3.
__device__ __forceinline__ float act_lo(int kind) { return kind == 0 ? -__builtin_huge_valf() : 0.0f; }
__device__ __forceinline__ float act_hi(int kind) { return kind == 2 ? 6.0f : __builtin_huge_valf(); }
__device__ __forceinline__ float clamp_act(float v, float lo, float hi) {
    return __builtin_amdgcn_fmed3f(v, lo, hi);
}
__device__ __forceinline__ float activate(float v, int kind) {
    return clamp_act(v, act_lo(kind), act_hi(kind));
}

// ------------------------------------------------------------------- K1 mask
// One lane per position: an fp32 fused multiply-add chain over the channels in
// ascending order from +0, then the bias, then the strict threshold m > 0.
template <typename T>
__global__ void __launch_bounds__(kBlock)
k_mask(const T *__restrict__ x, int64_t npix, int C, const float *__restrict__ w_m, float b_m,
       uint8_t *__restrict__ mask, float *__restrict__ logits) {
    int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i >= npix) return;
    const T *row = x + i * C;
    float acc = 0.0f;
    for (int c0 = 0; c0 < C; c0 += 8) {
        float v[8];
        io<T>::load8(row + c0, v);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = __builtin_fmaf(w_m[c0 + u], v[u], acc);
    }
    float m = acc + b_m;
    mask[i] = (m > 0.0f) ? 1 : 0;
    if (logits) logits[i] = m;
}

// ------------------------------------------------------ K2 bookkeeping helpers
__device__ __forceinline__ bool dilated_at(const uint8_t *__restrict__ mask, int n, int h, int w,
                                           int H, int W, int r) {
    bool d = false;
    for (int dh = -r; dh <= r; ++dh) {
        int hh = h + dh;
        if (hh < 0 || hh >= H) continue;
        const uint8_t *mrow = mask + (static_cast<int64_t>(n) * H + hh) * W;
        for (int dw = -r; dw <= r; ++dw) {
            int ww = w + dw;
            if (ww >= 0 && ww < W && mrow[ww]) d = true;
        }
    }
    return d;
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
    return (lane == 0) ? 0ull : (~0ull >> (64 - lane));
}

// K2a: one wave per image row (row = n*H + h): counts of active and dilated
// positions, from 64-lane ballots.
__global__ void __launch_bounds__(kBlock)
k_rowcount(const uint8_t *__restrict__ mask, int N, int H, int W, int r, int2 *__restrict__ rowcnt) {
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave;
    if (row >= static_cast<int64_t>(N) * H) return;  // uniform per wave
    const int n = static_cast<int>(row / H), h = static_cast<int>(row % H);
    int ca = 0, cd = 0;
    for (int w0 = 0; w0 < W; w0 += kWave) {
        const int w = w0 + lane;
        bool a = false, d = false;
        if (w < W) {
            a = mask[row * W + w] != 0;
            d = dilated_at(mask, n, h, w, H, W, r);
        }
        ca += __popcll(__ballot(a));
        cd += __popcll(__ballot(d));
    }
    if (lane == 0) rowcnt[row] = make_int2(ca, cd);
}

// K2b: one workgroup of 1024 lanes; lane t owns a contiguous run of rows.
// rowoff[r] = (active, dilated) positions before row r; rowoff[nrows] and
// counts hold the totals P, P_d.
constexpr int kScanThreads = 1024;
__global__ void __launch_bounds__(kScanThreads)
k_rowscan(const int2 *__restrict__ rowcnt, int64_t nrows, int2 *__restrict__ rowoff,
          int32_t *__restrict__ counts) {
    __shared__ int2 part[kScanThreads];
    const int t = threadIdx.x;
    const int64_t per = (nrows + kScanThreads - 1) / kScanThreads;
    const int64_t r0 = t * per;
    const int64_t r1 = (r0 + per < nrows) ? r0 + per : nrows;
    int sa = 0, sd = 0;
    for (int64_t r = r0; r < r1; ++r) {
        int2 v = rowcnt[r];
        sa += v.x;
        sd += v.y;
    }
    part[t] = make_int2(sa, sd);
    __syncthreads();
    for (int off = 1; off < kScanThreads; off <<= 1) {
        int2 v = part[t];
        int2 u = (t >= off) ? part[t - off] : make_int2(0, 0);
        __syncthreads();
        part[t] = make_int2(v.x + u.x, v.y + u.y);
        __syncthreads();
    }
    int a = (t == 0) ? 0 : part[t - 1].x;
    int d = (t == 0) ? 0 : part[t - 1].y;
    for (int64_t r = r0; r < r1; ++r) {
        rowoff[r] = make_int2(a, d);
        int2 v = rowcnt[r];
        a += v.x;
        d += v.y;
    }
    if (t == kScanThreads - 1) {
        rowoff[nrows] = part[t];
        counts[0] = part[t].x;
        counts[1] = part[t].y;
    }
}

// K2c: one wave per image row.  The wave first records, for rows h-1, h and
// h+1, the dilated-mask ballot words of every 64-column segment and their
// running counts (LDS); then the active and dilated positions of row h get
// their ranks from ballots, and every active position looks up its 9
// neighbours' ranks among the dilated positions of the three rows.
__global__ void __launch_bounds__(kBlock)
k_compact(const uint8_t *__restrict__ mask, int N, int H, int W, int r,
          const int2 *__restrict__ rowoff, int32_t *__restrict__ active,
          int32_t *__restrict__ dilated, int32_t *__restrict__ nbr) {
    __shared__ uint64_t words[kWavesPerBlock][3][kMaxSeg];
    __shared__ int segpre[kWavesPerBlock][3][kMaxSeg];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave;
    const bool live = row < static_cast<int64_t>(N) * H;  // uniform per wave
    const int n = live ? static_cast<int>(row / H) : 0;
    const int h = live ? static_cast<int>(row % H) : 0;
    const int nseg = (W + kWave - 1) / kWave;

    if (live) {
        for (int q = 0; q < 3; ++q) {
            const int hh = h + q - 1;
            int pre = 0;
            for (int seg = 0; seg < nseg; ++seg) {
                const int w = seg * kWave + lane;
                bool d = false;
                if (hh >= 0 && hh < H && w < W) d = dilated_at(mask, n, hh, w, H, W, r);
                const uint64_t b = __ballot(d);
                if (lane == 0) {
                    words[wave][q][seg] = b;
                    segpre[wave][q][seg] = pre;
                }
                pre += __popcll(b);
            }
        }
    }
    __syncthreads();
    if (!live) return;

    const int2 base = rowoff[row];
    const uint64_t lt = lanemask_lt(lane);
    int pre_a = 0;
    for (int seg = 0; seg < nseg; ++seg) {
        const int w = seg * kWave + lane;
        const bool a = (w < W) && mask[row * W + w] != 0;
        const uint64_t ba = __ballot(a);
        const uint64_t bd = words[wave][1][seg];
        const int64_t pix = row * W + w;
        if ((bd >> lane) & 1ull) {
            dilated[base.y + segpre[wave][1][seg] + __popcll(bd & lt)] = static_cast<int32_t>(pix);
        }
        if (a) {
            const int64_t p = base.x + pre_a + __popcll(ba & lt);
            active[p] = static_cast<int32_t>(pix);
            int32_t *out = nbr + p * 9;
#pragma unroll
            for (int k = 0; k < 9; ++k) {
                const int dh = k / 3 - 1, dw = k % 3 - 1;
                const int hh = h + dh, ww = w + dw;
                int32_t j = -1;
                if (hh >= 0 && hh < H && ww >= 0 && ww < W) {
                    const int q = dh + 1, sg = ww / kWave, bit = ww % kWave;
                    const uint64_t wd = words[wave][q][sg];
                    if ((wd >> bit) & 1ull) {
                        const uint64_t below = (bit == 0) ? 0ull : (wd & (~0ull >> (64 - bit)));
                        j = rowoff[row + dh].y + segpre[wave][q][sg] + __popcll(below);
                    }
                }
                out[k] = j;
            }
        }
        pre_a += __popcll(ba);
    }
}

// ----------------------------------------------- K3+K4 gather + 1x1 expansion
// Each wave owns tiles of 16 rows of the intermediate tensor.  The rows' input
// pixels (dilated[j], or j itself when dense) are loaded straight into the
// B operand (16 bytes per lane), so the gather costs no extra pass.  For each
// 16-channel slice of the hidden layer the wave runs the C-long contraction
// on the matrix cores (D^T = W1 T^T: hidden channels along M, rows along N),
// adds the bias, applies the activation and stores 4 consecutive channels per
// lane.  MAXKS = ceil(C / 32) slices of the contraction stay in registers.
template <typename T, bool DENSE, int MAXKS>
__global__ void __launch_bounds__(kBlock)
k_expand(const T *__restrict__ x, int C, int E, const T *__restrict__ w1,
         const float *__restrict__ b1, int act1, const int32_t *__restrict__ dil,
         const int32_t *__restrict__ counts, int64_t dense_rows, T *__restrict__ h1) {
    typedef mma<T> M;
    // sparse: P_d from the device, clamped to the capacity N*H*W (= dense_rows)
    const int64_t nrows = DENSE ? dense_rows : min(max(static_cast<int64_t>(counts[1]), int64_t{0}), dense_rows);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const int64_t ntiles = (nrows + 15) / 16;
    const int nks = (C + 31) / 32;
    const int nmt = E / 16;
    // row dense_rows (one past the capacity) stays zero: the depthwise reads it
    // for neighbours outside the image or the dilated list
    if (blockIdx.x == 0)
        for (int e = threadIdx.x; e < E; e += kBlock) h1[dense_rows * E + e] = static_cast<T>(0.0f);
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave; t < ntiles;
         t += static_cast<int64_t>(gridDim.x) * kWavesPerBlock) {
        const int64_t j = t * 16 + r;
        const bool valid = j < nrows;
        const int64_t pix = valid ? (DENSE ? j : static_cast<int64_t>(dil[j])) : 0;
        typename M::frag b[MAXKS];
#pragma unroll
        for (int ks = 0; ks < MAXKS; ++ks) {
            const int c0 = ks * 32 + g * 8;
            b[ks] = (ks < nks && valid && c0 < C) ? M::load(x + pix * C + c0) : M::zero();
        }
        for (int mt = 0; mt < nmt; ++mt) {
            const int e = mt * 16 + r;
            const int e0 = mt * 16 + 4 * g;
            floatx4 acc = {b1[e0], b1[e0 + 1], b1[e0 + 2], b1[e0 + 3]};  // bias first
            // Every MFMA is issued unconditionally (slices past C get zero
            // fragments): a branch around an MFMA whose result is read at the
            // join has been compiled without the wait states the read needs.
#pragma unroll
            for (int ks = 0; ks < MAXKS; ++ks) {
                const int c0 = ks * 32 + g * 8;
                typename M::frag a = (ks < nks && c0 < C)
                    ? M::load(w1 + static_cast<int64_t>(e) * C + c0) : M::zero();
                acc = M::run(a, b[ks], acc);
            }
            if (valid) {
                float o[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = activate(acc[v], act1);
                io<T>::store4(h1 + j * E + e0, o);
            }
        }
    }
}

// ------------------------- K5+K6 depthwise + 1x1 projection + scatter-add
// Each wave owns tiles of 16 active rows.  Lane (r, g) computes the depthwise
// output of row r for the 8 hidden channels it supplies to the projection's B
// operand: 9 taps, each a 16-byte load of an expanded row found through the
// neighbour table (missing neighbours read the all-zero row N*H*W of the
// expanded tensor, so the loads carry no branch), fp32 accumulation with the
// folded depthwise weights staged transposed in LDS, bias, activation, rounding
// to the storage type.  The projection (F^T = W3 H2^T) accumulates over the
// hidden channels on the matrix cores; the epilogue adds bias and the identity
// path and writes y at the active position (in place when y == x).
template <typename T, bool DENSE, int MAXMT>
__global__ void __launch_bounds__(kBlock)
k_dw_project(const T *__restrict__ h1, const T *x, T *y, int N, int H, int W, int C, int E,
             const T *__restrict__ w2, const float *__restrict__ b2, int act2,
             const T *__restrict__ w3, const float *__restrict__ b3, int act3,
             const int32_t *__restrict__ act_list, const int32_t *__restrict__ nbr,
             const int32_t *__restrict__ counts) {
    typedef mma<T> M;
    extern __shared__ float lds[];  // [9][E] depthwise weights, then [E] bias
    for (int i = threadIdx.x; i < 9 * E; i += kBlock) {
        const int e = i / 9, k = i % 9;
        lds[k * E + e] = static_cast<float>(w2[i]);
    }
    for (int e = threadIdx.x; e < E; e += kBlock) lds[9 * E + e] = b2[e];
    __syncthreads();

    const int64_t HW = static_cast<int64_t>(H) * W;
    const int64_t npos = static_cast<int64_t>(N) * HW;
    // sparse: P from the device, clamped to the capacity N*H*W
    const int64_t nrows = DENSE ? npos : min(max(static_cast<int64_t>(counts[0]), int64_t{0}), npos);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const int64_t ntiles = (nrows + 15) / 16;
    const int nks = (E + 31) / 32;
    const int nmt = (C + 15) / 16;
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave; t < ntiles;
         t += static_cast<int64_t>(gridDim.x) * kWavesPerBlock) {
        const int64_t p = t * 16 + r;
        const bool valid = p < nrows;
        int64_t pix = 0;
        int32_t nb[9];
        if (DENSE) {
            pix = valid ? p : 0;
            const int hh0 = static_cast<int>((pix / W) % H), ww0 = static_cast<int>(pix % W);
#pragma unroll
            for (int k = 0; k < 9; ++k) {
                const int dh = k / 3 - 1, dw = k % 3 - 1;
                const bool in = valid && hh0 + dh >= 0 && hh0 + dh < H && ww0 + dw >= 0 && ww0 + dw < W;
                nb[k] = in ? static_cast<int32_t>(pix + dh * W + dw) : static_cast<int32_t>(npos);
            }
        } else {
            pix = valid ? static_cast<int64_t>(act_list[p]) : 0;
#pragma unroll
            for (int k = 0; k < 9; ++k) {
                const int32_t q = valid ? nbr[p * 9 + k] : -1;
                nb[k] = (q >= 0) ? q : static_cast<int32_t>(npos);  // missing: the zero row
            }
        }
        floatx4 acc[MAXMT];  // projection bias first
#pragma unroll
        for (int mt = 0; mt < MAXMT; ++mt) {
            const int c0 = mt * 16 + 4 * g;
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[mt][v] = (mt < nmt && c0 < C) ? b3[c0 + v] : 0.0f;
        }

        for (int ks = 0; ks < nks; ++ks) {
            const int e0 = ks * 32 + g * 8;
            const bool ein = e0 < E;
            float hv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) hv[u] = 0.0f;
            if (ein && valid) {
                float s[8];  // depthwise bias first, then the taps in order
#pragma unroll
                for (int u = 0; u < 8; ++u) s[u] = lds[9 * E + e0 + u];
#pragma unroll
                for (int k = 0; k < 9; ++k) {  // branch free: missing taps read zeros
                    float v[8];
                    io<T>::load8(h1 + static_cast<int64_t>(nb[k]) * E + e0, v);
                    const float *wk = lds + k * E + e0;
#pragma unroll
                    for (int u = 0; u < 8; ++u) s[u] = __builtin_fmaf(wk[u], v[u], s[u]);
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) hv[u] = activate(s[u], act2);
            }
            const typename M::frag bf = M::pack(hv);
#pragma unroll
            for (int mt = 0; mt < MAXMT; ++mt) {  // unconditional MFMAs, as in k_expand
                const int c = mt * 16 + r;
                typename M::frag a = (mt < nmt && ein && c < C)
                    ? M::load(w3 + static_cast<int64_t>(c) * E + e0) : M::zero();
                acc[mt] = M::run(a, bf, acc[mt]);
            }
        }
        if (valid) {
#pragma unroll
            for (int mt = 0; mt < MAXMT; ++mt) {
                const int c0 = mt * 16 + 4 * g;
                if (mt < nmt && c0 < C) {
                    float xv[4], o[4];
                    io<T>::load4(x + pix * C + c0, xv);
#pragma unroll
                    for (int v = 0; v < 4; ++v) o[v] = xv[v] + activate(acc[mt][v], act3);
                    io<T>::store4(y + pix * C + c0, o);
                }
            }
        }
    }
}

// Plain 16-byte copy (y != x: inactive positions keep x).
__global__ void __launch_bounds__(kBlock)
k_copy16(const uint4 *__restrict__ src, uint4 *__restrict__ dst, int64_t n16) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n16;
         i += static_cast<int64_t>(gridDim.x) * kBlock)
        dst[i] = src[i];
}

}  // namespace dynconv
