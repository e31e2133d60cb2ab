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
// Hard decision of the mask unit at inference.  mode 0 (G-Binary, Eq. 8 with
// the Gumbel noise fixed to zero): m > 0.  mode 1 (G-Softmax, Sec. 3.1.2):
// the probabilities of Eq. 6 and Eq. 7, sigmoid(m) and 1 - sigmoid(m), go
// through the Gumbel-Softmax of Eq. 5 at zero noise and tau = 1 (a softmax
// over their logarithms) and the position runs when the first class exceeds
// 1/2.  Both agree except where fp32 rounding decides, near m = 0.
__device__ __forceinline__ bool mask_decision(float m, int mode) {
    if (mode == 0) return m > 0.0f;
    const float p1 = 1.0f / (1.0f + expf(-m));
    const float p2 = 1.0f - p1;
    const float e1 = expf(logf(p1)), e2 = expf(logf(p2));
    return e1 / (e1 + e2) > 0.5f;
}

template <typename T>
__global__ void __launch_bounds__(kBlock)
k_mask(const T *__restrict__ x, int64_t npix, int C, const float *__restrict__ w_m, float b_m,
       uint8_t *__restrict__ mask, float *__restrict__ logits, int mode) {
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
    mask[i] = mask_decision(m, mode) ? 1 : 0;
    if (logits) logits[i] = m;
}

// ------------------------------------------------------ K2 bookkeeping helpers
__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
    return (lane == 0) ? 0ull : (~0ull >> (64 - lane));
}

// Bits of image columns seg*64 .. seg*64+63 that lie inside a row of width W.
__device__ __forceinline__ uint64_t seg_valid(int seg, int W) {
    const int n = W - seg * kWave;
    return (n >= kWave) ? ~0ull : ((1ull << n) - 1ull);
}

// Horizontal dilation by radius r of segment `seg` of one row, given the
// row's mask words (bit b of word s = column 64*s + b); columns past the
// neighbouring segments' edges come from those segments.
__device__ __forceinline__ uint64_t hdilate(const uint64_t *row, int seg, int nseg, int r, int W) {
    const uint64_t m = row[seg];
    const uint64_t lo = (seg > 0) ? row[seg - 1] : 0ull;
    const uint64_t hi = (seg + 1 < nseg) ? row[seg + 1] : 0ull;
    uint64_t d = m;
    for (int k = 1; k <= r; ++k) d |= (m << k) | (lo >> (kWave - k)) | (m >> k) | (hi << (kWave - k));
    return d & seg_valid(seg, W);
}

// K2a: one wave per image row (row = n*H + h): the row's mask words (ballots
// of 64 columns) and its counts of active and dilated positions (the 3x3
// (radius r) dilation: OR over rows h-r .. h+r of the horizontally dilated
// words).
__global__ void __launch_bounds__(kBlock)
k_rowcount(const uint8_t *__restrict__ mask, int N, int H, int W, int r, int2 *__restrict__ rowcnt,
           uint64_t *__restrict__ words) {
    __shared__ uint64_t rows[kWavesPerBlock][7][kMaxSeg];  // rows h-r .. h+r, r <= 3
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave;
    if (row >= static_cast<int64_t>(N) * H) return;  // uniform per wave; no block barrier below
    const int n = static_cast<int>(row / H), h = static_cast<int>(row % H);
    const int nseg = (W + kWave - 1) / kWave;
    for (int q = 0; q <= 2 * r; ++q) {
        const int hh = h + q - r;
        for (int seg = 0; seg < nseg; ++seg) {
            const int w = seg * kWave + lane;
            const bool a = hh >= 0 && hh < H && w < W && mask[(static_cast<int64_t>(n) * H + hh) * W + w] != 0;
            const uint64_t b = __ballot(a);
            if (lane == 0) rows[wave][q][seg] = b;
        }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    int ca = 0, cd = 0;
    for (int seg = lane; seg < nseg; seg += kWave) {
        uint64_t d = 0;
        for (int q = 0; q <= 2 * r; ++q) d |= hdilate(rows[wave][q], seg, nseg, r, W);
        const uint64_t m = rows[wave][r][seg];
        words[row * nseg + seg] = m;
        ca += __popcll(m);
        cd += __popcll(d);
    }
    for (int off = 32; off > 0; off >>= 1) {
        ca += __shfl_down(ca, off);
        cd += __shfl_down(cd, off);
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

// K2c: one wave per image row.  From the mask words of rows h-1-r .. h+1+r
// the wave forms the dilated words of rows h-1, h and h+1 and their running
// per-segment counts (LDS); then the active and dilated positions of row h
// get their ranks from the words, and every active position finds its 9
// neighbours' ranks among the dilated positions of the three rows.
__global__ void __launch_bounds__(kBlock)
k_compact(const uint64_t *__restrict__ words, int N, int H, int W, int r,
          const int2 *__restrict__ rowoff, int32_t *__restrict__ active,
          int32_t *__restrict__ dilated, int32_t *__restrict__ nbr) {
    __shared__ uint64_t dw[kWavesPerBlock][3][kMaxSeg];
    __shared__ int segpre[kWavesPerBlock][3][kMaxSeg];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave;
    if (row >= static_cast<int64_t>(N) * H) return;  // uniform per wave; no block barrier below
    const int h = static_cast<int>(row % H);
    const int nseg = (W + kWave - 1) / kWave;

    // dilated words of rows h-1, h, h+1 (zero outside the image)
    for (int seg = lane; seg < nseg; seg += kWave) {
        for (int q = 0; q < 3; ++q) {
            const int hc = h + q - 1;
            uint64_t d = 0;
            if (hc >= 0 && hc < H) {
                for (int dh = -r; dh <= r; ++dh) {
                    const int hh = hc + dh;
                    if (hh < 0 || hh >= H) continue;
                    const uint64_t *wr = words + (row + (hh - h)) * nseg;
                    uint64_t m = wr[seg];
                    const uint64_t lo = (seg > 0) ? wr[seg - 1] : 0ull;
                    const uint64_t hi = (seg + 1 < nseg) ? wr[seg + 1] : 0ull;
                    uint64_t x = m;
                    for (int k = 1; k <= r; ++k)
                        x |= (m << k) | (lo >> (kWave - k)) | (m >> k) | (hi << (kWave - k));
                    d |= x;
                }
                d &= seg_valid(seg, W);
            }
            dw[wave][q][seg] = d;
        }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    if (lane < 3) {  // running counts per segment of rows h-1, h, h+1
        int pre = 0;
        for (int seg = 0; seg < nseg; ++seg) {
            segpre[wave][lane][seg] = pre;
            pre += __popcll(dw[wave][lane][seg]);
        }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");

    const int2 base = rowoff[row];
    const uint64_t lt = lanemask_lt(lane);
    int pre_a = 0;
    for (int seg = 0; seg < nseg; ++seg) {
        const int w = seg * kWave + lane;
        const uint64_t ba = words[row * nseg + seg];
        const uint64_t bd = dw[wave][1][seg];
        const int64_t pix = row * W + w;
        if ((bd >> lane) & 1ull)
            dilated[base.y + segpre[wave][1][seg] + __popcll(bd & lt)] = static_cast<int32_t>(pix);
        if ((ba >> lane) & 1ull) {
            const int64_t p = base.x + pre_a + __popcll(ba & lt);
            active[p] = static_cast<int32_t>(pix);
            int32_t *out = nbr + p * 9;
#pragma unroll
            for (int k = 0; k < 9; ++k) {
                const int dh = k / 3 - 1, dwc = k % 3 - 1;
                const int hh = h + dh, ww = w + dwc;
                int32_t j = -1;
                if (hh >= 0 && hh < H && ww >= 0 && ww < W) {
                    const int q = dh + 1, sg = ww / kWave, bit = ww % kWave;
                    const uint64_t wd = dw[wave][q][sg];
                    if ((wd >> bit) & 1ull) {
                        const uint64_t below = (bit == 0) ? 0ull : (wd & (~0ull >> (kWave - bit)));
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
// B operand (16 bytes per lane), so the gather costs no extra pass; the next
// tile's rows are requested before the current one is computed.  For each
// 16-channel slice of the hidden layer the wave runs the C-long contraction
// on the matrix cores (D^T = W1 T^T: hidden channels along M, rows along N),
// starting from the bias, applies the activation and stores 4 consecutive
// channels per lane.  With LDSW the expansion weights and bias are staged in
// LDS once per workgroup (row stride C+8); otherwise the A fragments come
// from memory.  MAXKS = ceil(C / 32) slices of the contraction.
template <typename T, bool DENSE, int MAXKS, bool LDSW>
__global__ void __launch_bounds__(kBlock)
k_expand(const T *__restrict__ x, int C, int E, const T *__restrict__ w1,
         const float *__restrict__ b1, int act1, const int32_t *__restrict__ dil,
         const int32_t *__restrict__ counts, int64_t dense_rows, T *__restrict__ h1, int eslab,
         int grid_per_slab) {
    typedef mma<T> M;
    extern __shared__ __align__(16) unsigned char ex_lds[];
    // sparse: P_d from the device, clamped to the capacity N*H*W (= dense_rows)
    const int64_t nrows = DENSE ? dense_rows : min(max(static_cast<int64_t>(counts[1]), int64_t{0}), dense_rows);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const int64_t ntiles = (nrows + 15) / 16;
    const int nks = (C + 31) / 32;
    // hidden channels e_base .. e_base + e_cnt - 1 (a slab whose expansion
    // weights fit in LDS; workgroups are grouped by slab)
    const int slab = blockIdx.x / grid_per_slab;
    const int bx = blockIdx.x % grid_per_slab;
    const int e_base = slab * eslab;
    const int e_cnt = min(eslab, E - e_base);
    const int nmt = e_cnt / 16;
    const float lo1 = act_lo(act1), hi1 = act_hi(act1);
    // row dense_rows (one past the capacity) stays zero: the depthwise reads it
    // for neighbours outside the image or the dilated list
    if (blockIdx.x == 0)
        for (int e = threadIdx.x; e < E; e += kBlock) h1[dense_rows * E + e] = static_cast<T>(0.0f);
    // XCD-aware order: workgroup i runs on XCD i % 8; each XCD walks its own
    // contiguous range of tiles (gridDim.x is a multiple of 8)
    const int64_t per_xcd = (ntiles + 7) / 8;
    const int64_t xcd = bx % 8, slot = bx / 8, nslot = grid_per_slab / 8;
    if (slot * kWavesPerBlock >= per_xcd) return;  // uniform per workgroup
    const int cs = C + 8;  // LDS row stride of the weights
    T *w1s = reinterpret_cast<T *>(ex_lds);
    float *b1s = reinterpret_cast<float *>(ex_lds + ((static_cast<size_t>(e_cnt) * cs * sizeof(T) + 15) & ~size_t(15)));
    if (LDSW) {
        constexpr int per16 = 16 / static_cast<int>(sizeof(T));
        const int vpr = C / per16;
        for (int i = threadIdx.x; i < e_cnt * vpr; i += kBlock) {
            const int e = i / vpr, k = i % vpr;
            *reinterpret_cast<uint4 *>(w1s + e * cs + k * per16) =
                *reinterpret_cast<const uint4 *>(w1 + static_cast<int64_t>(e_base + e) * C + k * per16);
        }
        for (int e = threadIdx.x; e < e_cnt; e += kBlock) b1s[e] = b1[e_base + e];
        __syncthreads();
    }
    const int64_t stride = nslot * kWavesPerBlock;  // in tiles of this XCD's range
    const int64_t t_end = min((xcd + 1) * per_xcd, ntiles);
    auto load_rows = [&](int64_t t, typename M::frag (&b)[MAXKS]) {
        const int64_t j = t * 16 + r;
        const bool valid = t < t_end && j < nrows;
        const int64_t pix = valid ? (DENSE ? j : static_cast<int64_t>(dil[j])) : 0;
#pragma unroll
        for (int ks = 0; ks < MAXKS; ++ks) {
            const int c0 = ks * 32 + g * 8;
            b[ks] = (ks < nks && valid && c0 < C) ? M::load(x + pix * C + c0) : M::zero();
        }
    };
    int64_t t = xcd * per_xcd + slot * kWavesPerBlock + wave;
    typename M::frag b[MAXKS];
    load_rows(t, b);
    for (; t < t_end; t += stride) {
        typename M::frag bn[MAXKS];
        load_rows(t + stride, bn);  // next tile's rows in flight meanwhile
        const int64_t j = t * 16 + r;
        const bool valid = j < nrows;
        for (int mt = 0; mt < nmt; ++mt) {
            const int el = mt * 16 + r;           // slab-local A row
            const int e = e_base + el;
            const int e0l = mt * 16 + 4 * g;      // slab-local output channel
            const int e0 = e_base + e0l;
            floatx4 acc;  // bias first
            if (LDSW) {
                acc = *reinterpret_cast<const floatx4 *>(b1s + e0l);
            } else {
                acc = floatx4{b1[e0], b1[e0 + 1], b1[e0 + 2], b1[e0 + 3]};
            }
            // Every MFMA is issued unconditionally (slices past C get zero
            // fragments): a branch around an MFMA whose result is read at the
            // join has been compiled without the wait states the read needs.
#pragma unroll
            for (int ks = 0; ks < MAXKS; ++ks) {
                const int c0 = ks * 32 + g * 8;
                typename M::frag a;
                if (LDSW)
                    a = (ks < nks && c0 < C) ? M::load(w1s + el * cs + c0) : M::zero();
                else
                    a = (ks < nks && c0 < C) ? M::load(w1 + static_cast<int64_t>(e) * C + c0) : M::zero();
                acc = M::run(a, b[ks], acc);
            }
            if (valid) {
                float o[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = clamp_act(acc[v], lo1, hi1);
                io<T>::store4(h1 + j * E + e0, o);
            }
        }
#pragma unroll
        for (int ks = 0; ks < MAXKS; ++ks) b[ks] = bn[ks];
    }
}

// ------------------------- K5+K6 depthwise + 1x1 projection + scatter-add
// A workgroup takes groups of kDwGroup tiles of 16 active rows.  The
// depthwise of one tile for one 32-channel slice of the hidden layer is a
// work item; the items of a group are spread over the four waves: lane (r, g)
// computes the depthwise output of row r for the 8 hidden channels it would
// supply to the projection's B operand (9 taps, each a 16-byte load of an
// expanded row found through the neighbour table -- missing neighbours read
// the all-zero row N*H*W -- fp32 accumulation from the bias with the folded
// weights staged transposed in LDS, activation, rounding to the storage
// type) and parks that fragment in LDS.  Then one wave per tile runs the
// projection (F^T = W3 H2^T) over the slices in order on the matrix cores,
// starting from the projection bias, and the epilogue adds the identity path
// and writes y at the active position (in place when y == x).  Hidden slices
// pass through LDS in chunks of kDwChunk.
// With SLABS the output channels are cut into nos slabs of MAXMT 16-row tiles; a work
// item is (group, slab).  Every slab of a group recomputes the group's
// depthwise (identical values) and projects onto its own output rows, so
// small images with many channels (7x7x160, 960 hidden) still spread over
// the chip; each output keeps one accumulator chain, in the same order.
constexpr int kDwGroup = 2;
constexpr int kDwChunk = 8;

constexpr int kDwChunkCh = kDwChunk * 32;  // hidden channels per chunk

template <typename T>
__host__ __device__ constexpr size_t dw_lds_bytes() {
    return 9 * kDwChunkCh * sizeof(T)                                      // w2 of a chunk, [9][256]
           + 4 * kDwChunkCh                                                // b2 of a chunk
           + static_cast<size_t>(kDwGroup) * kDwChunk * kWave * sizeof(typename mma<T>::frag)  // fragments
           + static_cast<size_t>(kDwGroup) * 16 * 10 * 4;                 // positions + neighbour rows
}

template <typename T, bool DENSE, int MAXMT, bool SLABS>
__global__ void __launch_bounds__(kBlock)
k_dw_project(const T *__restrict__ h1, const T *x, T *y, int N, int H, int W, int C, int E,
             const T *__restrict__ w2, const float *__restrict__ b2, int act2,
             const T *__restrict__ w3, const float *__restrict__ b3, int act3,
             const int32_t *__restrict__ act_list, const int32_t *__restrict__ nbr,
             const int32_t *__restrict__ counts, int nos_arg) {
    typedef mma<T> M;
    typedef typename M::frag Frag;
    extern __shared__ __align__(16) unsigned char dw_lds[];
    const int64_t HW = static_cast<int64_t>(H) * W;
    const int64_t npos = static_cast<int64_t>(N) * HW;
    // sparse: P from the device, clamped to the capacity N*H*W
    const int64_t nrows = DENSE ? npos : min(max(static_cast<int64_t>(counts[0]), int64_t{0}), npos);
    constexpr int GR = kDwGroup * 16;  // rows per group
    const int64_t ngroups = (nrows + GR - 1) / GR;
    // workgroup b: XCD b % 8, output slab (b / 8) % nos, group slot (b / 8) / nos
    // (without SLABS one slab: the register budget of the common case stays
    // that of a kernel without slab arithmetic)
    const int nos = SLABS ? nos_arg : 1;
    const int os = SLABS ? static_cast<int>((blockIdx.x / 8) % nos) : 0;
    const int mt0 = os * MAXMT;  // first output tile of the slab
    if ((blockIdx.x / 8) / nos >= (ngroups + 7) / 8) return;  // no group on this slot (uniform)
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const int nsl = (E + 31) / 32;
    const int nmt = (C + 15) / 16;
    const float lo2 = act_lo(act2), hi2 = act_hi(act2);
    const float lo3 = act_lo(act3), hi3 = act_hi(act3);

    T *w2t = reinterpret_cast<T *>(dw_lds);  // [9][kDwChunkCh]: the chunk's taps, transposed
    size_t off = 9 * kDwChunkCh * sizeof(T);
    float *b2s = reinterpret_cast<float *>(dw_lds + off);
    off += 4 * kDwChunkCh;
    Frag *fr = reinterpret_cast<Frag *>(dw_lds + off);  // [kDwGroup][kDwChunk][64]
    off += static_cast<size_t>(kDwGroup) * kDwChunk * kWave * sizeof(Frag);
    int32_t *gpix = reinterpret_cast<int32_t *>(dw_lds + off);  // [GR]
    int32_t *gnb = gpix + GR;                                   // [GR][9]
    // depthwise weights and bias of hidden channels e_base .. e_base+255
    auto stage_chunk = [&](int e_base) {
        const int ne = min(kDwChunkCh, E - e_base);
        for (int i = threadIdx.x; i < 9 * ne; i += kBlock) {
            const int e = i / 9, k = i % 9;
            w2t[k * kDwChunkCh + e] = w2[static_cast<int64_t>(e_base) * 9 + i];
        }
        for (int e = threadIdx.x; e < ne; e += kBlock) b2s[e] = b2[e_base + e];
    };
    const bool one_chunk = nsl <= kDwChunk;
    if (one_chunk) stage_chunk(0);  // visible after the group's first barrier

    // XCD-aware order: workgroup i runs on XCD i % 8; each XCD walks its own
    // contiguous range of groups, so the rows a group's taps read (the
    // previous and next image rows) were just expanded or read on that XCD
    // and sit in its L2; the slabs of a group run on the same XCD.
    // gridDim.x is a multiple of 8 * nos.
    const int64_t per_xcd = (ngroups + 7) / 8;
    const int64_t xcd = blockIdx.x % 8, slot = (blockIdx.x / 8) / nos, nslot = gridDim.x / 8 / nos;
    for (int64_t k = slot; k < per_xcd; k += nslot) {
        const int64_t grp = xcd * per_xcd + k;
        if (grp >= ngroups) break;  // uniform per workgroup
        const int64_t p0 = grp * GR;
        const int gt = static_cast<int>(min(static_cast<int64_t>(kDwGroup), (nrows - p0 + 15) / 16));
        // positions and neighbour rows of the group (missing: the zero row)
        for (int i = threadIdx.x; i < GR; i += kBlock) {
            const int64_t p = p0 + i;
            const bool valid = p < nrows;
            const int64_t pix = valid ? (DENSE ? p : static_cast<int64_t>(act_list[p])) : -1;
            gpix[i] = static_cast<int32_t>(pix);
            if (DENSE) {
                const int hh0 = valid ? static_cast<int>((pix / W) % H) : 0;
                const int ww0 = valid ? static_cast<int>(pix % W) : 0;
#pragma unroll
                for (int k = 0; k < 9; ++k) {
                    const int dh = k / 3 - 1, dwc = k % 3 - 1;
                    const bool in = valid && hh0 + dh >= 0 && hh0 + dh < H && ww0 + dwc >= 0 && ww0 + dwc < W;
                    gnb[i * 9 + k] = in ? static_cast<int32_t>(pix + dh * W + dwc) : static_cast<int32_t>(npos);
                }
            } else {
#pragma unroll
                for (int k = 0; k < 9; ++k) {
                    const int32_t q = valid ? nbr[p * 9 + k] : -1;
                    gnb[i * 9 + k] = (q >= 0) ? q : static_cast<int32_t>(npos);
                }
            }
        }
        __syncthreads();
        // the projection wave's tile (waves past the group's tiles repeat the
        // last one, so every wave issues the same MFMAs; only real tiles store)
        const int pt = min(wave, gt - 1);
        floatx4 acc[MAXMT];  // projection bias first
#pragma unroll
        for (int mt = 0; mt < MAXMT; ++mt) {
            const int c0 = (mt0 + mt) * 16 + 4 * g;
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[mt][v] = (mt0 + mt < nmt && c0 < C) ? b3[c0 + v] : 0.0f;
        }
        for (int s0 = 0; s0 < nsl; s0 += kDwChunk) {
            const int ns = min(kDwChunk, nsl - s0);
            if (!one_chunk) {
                stage_chunk(s0 * 32);
                __syncthreads();
            }
            // depthwise items (tile, slice) of this chunk
            for (int it = wave; it < gt * ns; it += kWavesPerBlock) {
                const int t = it % gt, sl = it / gt;
                const int q = t * 16 + r;
                const int e0 = (s0 + sl) * 32 + g * 8;
                float hv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) hv[u] = 0.0f;
                if (e0 < E && gpix[q] >= 0) {
                    const int el = e0 - s0 * 32;  // channel within the chunk
                    typename io<T>::vec8 tv[9];
#pragma unroll
                    for (int k = 0; k < 9; ++k)  // branch free: missing taps read zeros
                        tv[k] = io<T>::raw8(h1 + static_cast<int64_t>(gnb[q * 9 + k]) * E + e0);
                    float sacc[8];  // depthwise bias first, then the taps in order
#pragma unroll
                    for (int u = 0; u < 8; ++u) sacc[u] = b2s[el + u];
#pragma unroll
                    for (int k = 0; k < 9; ++k) {
                        const typename io<T>::vec8 wk = io<T>::raw8(w2t + k * kDwChunkCh + el);
#pragma unroll
                        for (int u = 0; u < 8; ++u)
                            sacc[u] = __builtin_fmaf(static_cast<float>(wk[u]), static_cast<float>(tv[k][u]), sacc[u]);
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) hv[u] = clamp_act(sacc[u], lo2, hi2);
                }
                fr[(t * kDwChunk + sl) * kWave + lane] = M::pack(hv);
            }
            __syncthreads();
            for (int sl = 0; sl < ns; ++sl) {
                const Frag bf = fr[(pt * kDwChunk + sl) * kWave + lane];
                const int e0 = (s0 + sl) * 32 + g * 8;
#pragma unroll
                for (int mt = 0; mt < MAXMT; ++mt) {  // unconditional MFMAs, as in k_expand
                    const int c = (mt0 + mt) * 16 + r;
                    const Frag a = (mt0 + mt < nmt && e0 < E && c < C)
                                       ? M::load(w3 + static_cast<int64_t>(c) * E + e0)
                                       : M::zero();
                    acc[mt] = M::run(a, bf, acc[mt]);
                }
            }
            __syncthreads();
        }
        const int64_t pix = gpix[pt * 16 + r];
        if (wave < gt && pix >= 0) {
#pragma unroll
            for (int mt = 0; mt < MAXMT; ++mt) {
                const int c0 = (mt0 + mt) * 16 + 4 * g;
                if (mt0 + mt < nmt && c0 < C) {
                    float xv[4], o[4];
                    io<T>::load4(x + pix * C + c0, xv);
#pragma unroll
                    for (int v = 0; v < 4; ++v) o[v] = xv[v] + clamp_act(acc[mt][v], lo3, hi3);
                    io<T>::store4(y + pix * C + c0, o);
                }
            }
        }
        __syncthreads();  // gpix / gnb are rewritten for the next group
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
