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
// A work item is a tile of 64 positions (16 per wave) and a range of OT
// 16-row output tiles.  Outputs run along M (rows of w), positions along N:
// lane (r, g) supplies 8 consecutive channels of position r (B) and of output
// row r (A).  The contraction runs in chunks of KB 32-channel steps: the
// wave issues the chunk's KB x loads at once, the workgroup stages the
// chunk's weights for its output range in LDS (rows padded by 8 elements),
// then every wave runs KB x OT matrix-core steps from there.  With one chunk
// (C <= 32 KB) the weights are staged once per workgroup: a workgroup keeps
// its output range and walks position tiles, requesting the next tile's x
// before it contracts the current one.  The accumulation starts from
// the bias and takes c in ascending steps of 32, zero past C.  Every MFMA is
// issued unconditionally (zero fragments out of range).
// Workgroup b runs on XCD b % 8 and takes output range (b / 8) % nor; the
// nor workgroups of one position tile run on the same XCD, so its x rows
// are read from HBM once.
constexpr int kPwPos = 64;

template <typename T, int OT, int KB>
__host__ __device__ constexpr size_t pw_lds_bytes() {
    return static_cast<size_t>(OT) * 16 * (KB * 32 + 8) * sizeof(T);
}

template <typename T, int OT, int KB>
__global__ void __launch_bounds__(kBlock)
k_conv1x1(const T *__restrict__ x, int64_t P, int C, const T *__restrict__ w, const float *__restrict__ b,
          int O, int act, const T *__restrict__ res, T *__restrict__ y, int nor) {
    typedef mma<T> M;
    typedef typename M::frag Frag;
    constexpr int ROWS = OT * 16;
    constexpr int LD = KB * 32 + 8;  // LDS row pitch in elements
    constexpr int PIECES = KB * 4;   // 8-element pieces per staged row
    extern __shared__ __align__(16) unsigned char pw_lds[];
    T *ws = reinterpret_cast<T *>(pw_lds);  // [ROWS][LD]
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const int xcd = blockIdx.x % 8;
    const int orng = static_cast<int>((blockIdx.x / 8) % nor);
    const int64_t slot = (blockIdx.x / 8) / nor, nslot = gridDim.x / 8 / nor;
    const int o_base = orng * ROWS;
    const int64_t ptiles = (P + kPwPos - 1) / kPwPos;
    const int nch = (C + KB * 32 - 1) / (KB * 32);
    const float lo = act_lo(act), hi = act_hi(act);
    // weights of output rows o_base .. o_base+ROWS-1, channels c_base .. c_base+32KB-1
    auto stage = [&](int c_base) {
        for (int i = threadIdx.x; i < ROWS * PIECES; i += kBlock) {
            const int row = i / PIECES, c = c_base + (i % PIECES) * 8;
            const int o = o_base + row;
            const Frag v = (o < O && c < C) ? M::load(w + static_cast<int64_t>(o) * C + c) : M::zero();
            *reinterpret_cast<Frag *>(ws + row * LD + (c - c_base)) = v;
        }
    };
    auto init = [&](floatx4 (&acc)[OT]) {
#pragma unroll
        for (int mt = 0; mt < OT; ++mt) {
            const int o0 = o_base + mt * 16 + 4 * g;
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[mt][v] = (o0 + v < O) ? b[o0 + v] : 0.0f;
        }
    };
    auto load_x = [&](Frag (&bx)[KB], int64_t p, int c_base) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            const int c = c_base + kb * 32 + 8 * g;
            bx[kb] = (p < P && c < C) ? M::load(x + p * C + c) : M::zero();
        }
    };
    auto contract = [&](floatx4 (&acc)[OT], const Frag (&bx)[KB]) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
            for (int mt = 0; mt < OT; ++mt) {
                const Frag a = *reinterpret_cast<const Frag *>(ws + (mt * 16 + r) * LD + kb * 32 + 8 * g);
                acc[mt] = M::run(a, bx[kb], acc[mt]);
            }
        }
    };
    auto finish = [&](const floatx4 (&acc)[OT], int64_t p) {
#pragma unroll
        for (int mt = 0; mt < OT; ++mt) {
            const int o0 = o_base + mt * 16 + 4 * g;
            if (p < P && o0 < O) {  // O is a multiple of 8: all four outputs exist
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
    };
    const int64_t step = nslot * 8;
    const int64_t lane_p = wave * 16 + r;  // this lane's position within a tile (B column)
    if (nch == 1) {
        // weights staged once; the next tile's x is requested before the
        // current tile is contracted
        stage(0);
        __syncthreads();
        int64_t pt = slot * 8 + xcd;
        Frag bn[KB];
        load_x(bn, pt * kPwPos + lane_p, 0);
        for (; pt < ptiles; pt += step) {
            // small weight ranges stay in registers across tiles; larger ones
            // are re-read from LDS per tile (a compiler barrier keeps them
            // from being hoisted out of the loop)
            if constexpr (OT * KB * sizeof(Frag) > 128) __asm__ volatile("" ::: "memory");
            Frag bx[KB];
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) bx[kb] = bn[kb];
            if (pt + step < ptiles) load_x(bn, (pt + step) * kPwPos + lane_p, 0);
            floatx4 acc[OT];
            init(acc);
            contract(acc, bx);
            finish(acc, pt * kPwPos + lane_p);
        }
        return;
    }
    for (int64_t pt = slot * 8 + xcd; pt < ptiles; pt += step) {
        const int64_t p = pt * kPwPos + lane_p;
        floatx4 acc[OT];
        init(acc);
        for (int ch = 0; ch < nch; ++ch) {
            const int c_base = ch * KB * 32;
            Frag bx[KB];
            load_x(bx, p, c_base);
            __syncthreads();  // every wave is done with the previous chunk
            stage(c_base);
            __syncthreads();
            contract(acc, bx);
        }
        finish(acc, p);
    }
}

// ------------------------------------------------------------ depthwise
// A work item is (image, block of R output rows, 256 consecutive (column,
// 8-channel group) tasks, groups fastest).  A lane's task walks the input
// rows of its R output rows once: each input row's three taps (16-byte
// loads, zeros past the left and right edges) feed every output row that
// uses it, so a lane issues (S (R - 1) + 3) x 3 tap loads for R outputs
// instead of 9 R.  The 9 weight vectors are loaded once per task.  Each
// output accumulates in fp32 from the bias, taps in (kh, kw) order; rows
// outside the image are skipped.
template <typename T, int S, int R>
__global__ void __launch_bounds__(kBlock)
k_dwconv3x3(const T *__restrict__ x, int N, int H, int W, int C, const T *__restrict__ w,
            const float *__restrict__ b, int act, T *__restrict__ y, int Ho, int Wo) {
    typedef typename io<T>::vec8 V;
    constexpr int ROWS = S * (R - 1) + 3;  // input rows of R output rows
    extern __shared__ __align__(16) unsigned char dw_smem[];
    T *wt = reinterpret_cast<T *>(dw_smem);  // [9][C]: the taps, transposed
    for (int i = threadIdx.x; i < 9 * C; i += kBlock) {
        const int ch = i / 9, k = i % 9;
        wt[k * C + ch] = w[i];
    }
    __syncthreads();
    const float lo = act_lo(act), hi = act_hi(act);
    const int cgs = C / 8;
    const int tasks = Wo * cgs;
    const int chunks = (tasks + kBlock - 1) / kBlock;
    const int rbs = (Ho + R - 1) / R;
    const int64_t items = static_cast<int64_t>(N) * rbs * chunks;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int chunk = static_cast<int>(it % chunks);
        const int64_t nr = it / chunks;
        const int rb = static_cast<int>(nr % rbs), n = static_cast<int>(nr / rbs);
        const int task = chunk * kBlock + static_cast<int>(threadIdx.x);
        if (task >= tasks) continue;
        const int cg = task % cgs, j = task / cgs, c = cg * 8;
        const int i0 = rb * R;  // first output row
        V wk[9];
#pragma unroll
        for (int k = 0; k < 9; ++k) wk[k] = io<T>::raw8(wt + k * C + c);
        float acc[R][8];
#pragma unroll
        for (int q = 0; q < R; ++q)
#pragma unroll
            for (int u = 0; u < 8; ++u) acc[q][u] = b[c + u];
        const T *img = x + static_cast<int64_t>(n) * H * W * C;
#pragma unroll
        for (int t = 0; t < ROWS; ++t) {
            const int hh = S * i0 - 1 + t;
            if (hh < 0 || hh >= H) continue;
            V v[3];
#pragma unroll
            for (int dw = 0; dw < 3; ++dw) {
                const int ww = S * j - 1 + dw;
                if (ww >= 0 && ww < W) {
                    v[dw] = io<T>::raw8(img + (static_cast<int64_t>(hh) * W + ww) * C + c);
                } else {
                    v[dw] = V{};
                }
            }
#pragma unroll
            for (int q = 0; q < R; ++q) {
                const int dh = t - S * q;  // compile-time after unrolling
                if (dh < 0 || dh > 2) continue;
#pragma unroll
                for (int dw = 0; dw < 3; ++dw)
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        acc[q][u] = __builtin_fmaf(static_cast<float>(wk[dh * 3 + dw][u]),
                                                   static_cast<float>(v[dw][u]), acc[q][u]);
            }
        }
#pragma unroll
        for (int q = 0; q < R; ++q) {
            if (i0 + q >= Ho) break;
            float o[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) o[u] = clamp_act(acc[q][u], lo, hi);
            T *dst = y + ((static_cast<int64_t>(n) * Ho + i0 + q) * Wo + j) * C + c;
            io<T>::store4(dst, o);
            io<T>::store4(dst + 4, o + 4);
        }
    }
}

// ------------------------------------------------------ expansion + depthwise
// An ungated block's 1x1 expansion and depthwise 3x3 in one launch, so that
// the expanded tensor never goes to HBM.  A work item is a tile of 8 x 8
// depthwise outputs of one image; its input region, (S*7+3)^2 positions, is
// staged in LDS (rows of C + 8 elements, zeros outside the image).  The
// workgroups are persistent: each stages all weights in LDS once (expansion
// rows of C + 8, depthwise taps transposed to [9][E]) and walks items,
// loading the next item's region into registers while it computes the
// current one.  Per 32-channel slice of the hidden layer: each wave expands
// 16-position tiles of the region on the matrix cores (operands as in
// k_conv1x1: bias first, 32-channel steps ascending), applies the activation
// and stores the slice into a region array (zeros at positions outside the
// image: the depthwise's zero padding); then lane (o, cg) computes the
// depthwise of output o for 8 hidden channels from 9 fixed slots of that
// array, fp32 from the bias, taps in (kh, kw) order, and writes it to
// h2 [Ho*Wo][E].
constexpr int kEdTile = 8;  // depthwise outputs per tile side

template <int S>
__host__ __device__ constexpr int ed_region_side() { return S * (kEdTile - 1) + 3; }
template <int S>
__host__ __device__ constexpr int ed_region_tiles() {
    return (ed_region_side<S>() * ed_region_side<S>() + 15) / 16;
}
template <typename T, int S>
__host__ __device__ constexpr size_t ed_lds_bytes(int C, int E) {
    return static_cast<size_t>(ed_region_tiles<S>()) * 16 * ((C + 8) + 40) * sizeof(T)  // xs + h1
           + static_cast<size_t>(E) * (C + 8) * sizeof(T) + 9 * static_cast<size_t>(E) * sizeof(T)  // w1, w2t
           + 8 * static_cast<size_t>(E);                                                            // b1, b2
}

template <typename T, int S, int KS>
__global__ void __launch_bounds__(kBlock)
k_expand_dw(const T *__restrict__ x, int N, int H, int W, int C, const T *__restrict__ w1,
            const float *__restrict__ b1, int act1, int E, const T *__restrict__ w2, const float *__restrict__ b2,
            int act2, T *__restrict__ h2, int Ho, int Wo) {
    typedef mma<T> M;
    typedef typename M::frag Frag;
    typedef typename io<T>::vec8 V;
    constexpr int RS = ed_region_side<S>();
    constexpr int RP = RS * RS;
    constexpr int NT = ed_region_tiles<S>();
    constexpr int TPW = (NT + kWavesPerBlock - 1) / kWavesPerBlock;  // tiles per wave
    constexpr int HP = 40;                                          // h1 row pitch (32 + 8)
    constexpr int XP = (NT * 16 * KS * 4 + kBlock - 1) / kBlock;     // x pieces per thread (<= 32)
    static_assert(XP <= 32, "x pieces per thread exceed the validity mask");
    extern __shared__ __align__(16) unsigned char ed_smem[];
    const int PX = C + 8;  // row pitch of x and of the expansion weights
    T *xs = reinterpret_cast<T *>(ed_smem);  // [NT*16][PX]
    T *h1 = xs + NT * 16 * PX;               // [NT*16][HP]
    T *w1s = h1 + NT * 16 * HP;              // [E][PX]
    T *w2t = w1s + E * PX;                   // [9][E]
    float *b1s = reinterpret_cast<float *>(w2t + 9 * E);  // [E]
    float *b2s = b1s + E;                                 // [E]
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int r = lane % 16, g = lane / 16;
    const float lo1 = act_lo(act1), hi1 = act_hi(act1), lo2 = act_lo(act2), hi2 = act_hi(act2);
    const int tr = (Ho + kEdTile - 1) / kEdTile, tc = (Wo + kEdTile - 1) / kEdTile;
    const int64_t items = static_cast<int64_t>(N) * tr * tc;
    const int nsl = (E + 31) / 32;
    const int pieces = C / 8;  // 16-byte pieces of an x row
    if (static_cast<int64_t>(blockIdx.x) >= items) return;
    // all weights, once
    for (int i = tid; i < E * pieces; i += kBlock) {
        const int e = i / pieces, pc = (i % pieces) * 8;
        *reinterpret_cast<V *>(w1s + e * PX + pc) = io<T>::raw8(w1 + static_cast<int64_t>(e) * C + pc);
    }
    for (int i = tid; i < 9 * E; i += kBlock) {
        const int e = i / 9, k = i % 9;
        w2t[k * E + e] = w2[i];
    }
    for (int e = tid; e < E; e += kBlock) {
        b1s[e] = b1[e];
        b2s[e] = b2[e];
    }
    // the item's region origin; one thread's x pieces of it, into registers
    auto origin = [&](int64_t it, int &n, int &i0, int &j0) {
        n = static_cast<int>(it / (tr * tc));
        const int rem = static_cast<int>(it % (tr * tc));
        i0 = (rem / tc) * kEdTile;
        j0 = (rem % tc) * kEdTile;
    };
    // Loads are issued unconditionally (pieces outside the image read the
    // tensor's first piece) and replaced by zeros only when stored, so no
    // wait for them is needed before the current item's slices.
    auto load_x = [&](int64_t it, V (&xr)[XP], uint32_t &ok) {
        int n, i0, j0;
        origin(it, n, i0, j0);
        const int hb = S * i0 - 1, wb = S * j0 - 1;
        const T *img = x + static_cast<int64_t>(n) * H * W * C;
        ok = 0;
#pragma unroll
        for (int q = 0; q < XP; ++q) {
            const int i = tid + q * kBlock;
            const int slot = i / pieces, pc = (i % pieces) * 8;
            const int hh = hb + slot / RS, ww = wb + slot % RS;
            const bool in = i < NT * 16 * pieces && slot < RP && hh >= 0 && hh < H && ww >= 0 && ww < W;
            xr[q] = io<T>::raw8(in ? img + (static_cast<int64_t>(hh) * W + ww) * C + pc : x);
            ok |= static_cast<uint32_t>(in) << q;
        }
    };
    auto store_x = [&](const V (&xr)[XP], uint32_t ok) {
#pragma unroll
        for (int q = 0; q < XP; ++q) {
            const int i = tid + q * kBlock;
            if (i < NT * 16 * pieces)
                *reinterpret_cast<V *>(xs + (i / pieces) * PX + (i % pieces) * 8) = ((ok >> q) & 1u) ? xr[q] : V{};
        }
    };
    V xr[XP];
    uint32_t xok;
    int64_t it = blockIdx.x;
    load_x(it, xr, xok);
    store_x(xr, xok);
    __syncthreads();
    for (;;) {
        const int64_t next = it + gridDim.x;
        if (next < items) load_x(next, xr, xok);
        int n, i0, j0;
        origin(it, n, i0, j0);
        const int hb = S * i0 - 1, wb = S * j0 - 1;
        // the item's B fragments (region x) and in-image flags, kept for
        // every slice; waves past the last tile repeat it (same values), so
        // every wave issues the same MFMAs
        Frag bx[TPW][KS];
        uint32_t inside = 0;
#pragma unroll
        for (int jt = 0; jt < TPW; ++jt) {
            const int t = wave + kWavesPerBlock * jt;
            const int slot = (t < NT ? t : NT - 1) * 16 + r;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int c = ks * 32 + 8 * g;
                bx[jt][ks] = (c < C) ? *reinterpret_cast<const Frag *>(xs + slot * PX + c) : M::zero();
            }
            const int hh = hb + slot / RS, ww = wb + slot % RS;
            inside |= static_cast<uint32_t>(slot < RP && hh >= 0 && hh < H && ww >= 0 && ww < W) << jt;
        }
        for (int sl = 0; sl < nsl; ++sl) {
            const int e0 = sl * 32;
            // the slice's expansion rows (A) and biases, once per slice
            Frag a1[2][KS];
            floatx4 binit[2];
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const int er = e0 + m * 16 + r;  // A row: hidden channel
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const int c = ks * 32 + 8 * g;
                    a1[m][ks] = (er < E && c < C) ? *reinterpret_cast<const Frag *>(w1s + er * PX + c) : M::zero();
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int e = e0 + m * 16 + 4 * g + v;
                    binit[m][v] = (e < E) ? b1s[e] : 0.0f;
                }
            }
            // D[e][slot]: rows are hidden channels, columns region slots
#pragma unroll
            for (int jt = 0; jt < TPW; ++jt) {
                const int t = wave + kWavesPerBlock * jt;
                const int slot = (t < NT ? t : NT - 1) * 16 + r;
                const bool in = (inside >> jt) & 1u;
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    floatx4 d = binit[m];
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) d = M::run(a1[m][ks], bx[jt][ks], d);
                    if (t < NT) {
                        float o[4];
#pragma unroll
                        for (int v = 0; v < 4; ++v) o[v] = in ? clamp_act(d[v], lo1, hi1) : 0.0f;
                        io<T>::store4(h1 + slot * HP + m * 16 + 4 * g, o);
                    }
                }
            }
            __syncthreads();
            // depthwise: lane (o, cg), output o of the tile, channels 8cg..8cg+7
            {
                const int o = tid / 4, cg = tid % 4;
                const int oi = o / kEdTile, oj = o % kEdTile;
                const int e8 = e0 + 8 * cg;
                const int i = i0 + oi, j = j0 + oj;
                if (e8 < E) {
                    float acc[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) acc[u] = b2s[e8 + u];
#pragma unroll
                    for (int k = 0; k < 9; ++k) {
                        const int slot = (S * oi + k / 3) * RS + S * oj + k % 3;
                        const V v = io<T>::raw8(h1 + slot * HP + 8 * cg);
                        const V wk = io<T>::raw8(w2t + k * E + e8);
#pragma unroll
                        for (int u = 0; u < 8; ++u)
                            acc[u] = __builtin_fmaf(static_cast<float>(wk[u]), static_cast<float>(v[u]), acc[u]);
                    }
                    if (i < Ho && j < Wo) {
                        float out[8];
#pragma unroll
                        for (int u = 0; u < 8; ++u) out[u] = clamp_act(acc[u], lo2, hi2);
                        T *dst = h2 + ((static_cast<int64_t>(n) * Ho + i) * Wo + j) * E + e8;
                        io<T>::store4(dst, out);
                        io<T>::store4(dst + 4, out + 4);
                    }
                }
            }
            __syncthreads();  // h1 is rewritten by the next slice, xs by the next item
        }
        if (next >= items) break;
        store_x(xr, xok);
        __syncthreads();
        it = next;
    }
}

// ------------------------------------------------------------ full 3x3
// One lane per output position computing 32 outputs at a time; weights
// [O][Ci][3][3] and biases staged in LDS as fp32, reordered to [k][ci][o] so
// that the 32 weights of one tap and input channel are 8 broadcast 16-byte
// reads.  Ci is small (the stem's 3 input channels): a lane reads each of its
// 9 Ci input values once per 32 outputs.  Accumulation in fp32 from the
// bias, taps in (kh, kw) order, input channels ascending (dynamic shared
// memory: 9*Ci*O + O floats).
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
    const int64_t total = static_cast<int64_t>(N) * Ho * Wo;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < total;
         q += static_cast<int64_t>(gridDim.x) * kBlock) {
        const int64_t ni = q / Wo;
        const int j = static_cast<int>(q - ni * Wo);
        const int n = static_cast<int>(ni / Ho), i = static_cast<int>(ni - static_cast<int64_t>(n) * Ho);
        const T *img = x + static_cast<int64_t>(n) * H * W * Ci;
        for (int o0 = 0; o0 < O; o0 += 32) {
            const int ng = min(4, (O - o0) / 8);  // 8-output groups in this pass
            float s[32];
#pragma unroll
            for (int u = 0; u < 32; ++u) s[u] = (u / 8 < ng) ? bs[o0 + u] : 0.0f;
#pragma unroll
            for (int k = 0; k < 9; ++k) {
                const int hh = stride * i + k / 3 - 1, ww = stride * j + k % 3 - 1;
                if (hh < 0 || hh >= H || ww < 0 || ww >= W) continue;
                const T *px = img + (static_cast<int64_t>(hh) * W + ww) * Ci;
                for (int c = 0; c < Ci; ++c) {
                    const float v = static_cast<float>(px[c]);
                    const float *wr = ws + (k * Ci + c) * O + o0;
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        if (gq >= ng) break;
                        const float4 wa = *reinterpret_cast<const float4 *>(wr + 8 * gq);
                        const float4 wb = *reinterpret_cast<const float4 *>(wr + 8 * gq + 4);
                        const float wk[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
#pragma unroll
                        for (int u = 0; u < 8; ++u) s[8 * gq + u] = __builtin_fmaf(wk[u], v, s[8 * gq + u]);
                    }
                }
            }
            T *dst = y + q * O + o0;
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                if (gq >= ng) break;
                float o[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) o[u] = clamp_act(s[8 * gq + u], lo, hi);
                io<T>::store4(dst + 8 * gq, o);
                io<T>::store4(dst + 8 * gq + 4, o + 4);
            }
        }
    }
}

// ------------------------------------------------ full 3x3 on the matrix cores
// The same convolution as an implicit-im2col contraction for 16-bit
// storage: the contraction index runs over (tap, input channel) pairs,
// kk = k * Ci + c with tap k = 3 kh + kw, zero-padded to KS steps of 32.
// Outputs run along M, output positions along N: lane (r, g) gathers the 8
// input values kk = 32 ks + 8 g .. +7 of its position r (zeros outside the
// image and past 9 Ci) straight into its B fragment, the weights sit in LDS
// as [O][32 KS + 8] rows in kk order, and the wave walks the outputs in
// ranges of OT tiles of 16.  Accumulation from the bias in kk order (32 at a
// time on the matrix core); the taps' (dh, dw, c) per kk come from a small
// LDS table.  Dynamic shared memory: O (32 KS + 8) elements + 32 KS ints.
template <typename T, int KS, int OT>
__global__ void __launch_bounds__(kBlock)
k_conv3x3_mfma(const T *__restrict__ x, int N, int H, int W, int Ci, int stride, const T *__restrict__ w,
               const float *__restrict__ b, int O, int act, T *__restrict__ y, int Ho, int Wo) {
    typedef mma<T> M;
    typedef typename M::frag Frag;
    constexpr int KP = KS * 32 + 8;  // LDS row pitch of the weights
    extern __shared__ __align__(16) unsigned char c3_smem[];
    T *ws = reinterpret_cast<T *>(c3_smem);         // [O][KP]
    int *tap = reinterpret_cast<int *>(ws + O * KP);  // [32 KS]: (dh+1) | (dw+1) << 2 | c << 4, -1 past 9 Ci
    const int K = 9 * Ci;
    for (int i = threadIdx.x; i < O * KP; i += kBlock) {
        const int o = i / KP, kk = i % KP;
        ws[i] = (kk < K) ? w[(o * Ci + kk % Ci) * 9 + kk / Ci] : static_cast<T>(0.0f);
    }
    for (int kk = threadIdx.x; kk < 32 * KS; kk += kBlock) {
        const int k = kk / Ci, c = kk % Ci;
        tap[kk] = (kk < K) ? ((k / 3) | ((k % 3) << 2) | (c << 4)) : -1;
    }
    __syncthreads();
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r = lane % 16, g = lane / 16;
    const float lo = act_lo(act), hi = act_hi(act);
    const int64_t total = static_cast<int64_t>(N) * Ho * Wo;
    const int64_t tiles = (total + 63) / 64;
    const int nmt = (O + 15) / 16;
    for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
        const int64_t q = t * 64 + wave * 16 + r;  // this lane's output position (B column)
        const bool qin = q < total;
        const int64_t qq = qin ? q : 0;
        const int64_t ni = qq / Wo;
        const int j = static_cast<int>(qq - ni * Wo);
        const int n = static_cast<int>(ni / Ho), i = static_cast<int>(ni - static_cast<int64_t>(n) * Ho);
        const int h0 = stride * i - 1, w0 = stride * j - 1;
        const T *img = x + static_cast<int64_t>(n) * H * W * Ci;
        Frag bx[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int e = tap[ks * 32 + 8 * g + u];
                const int hh = h0 + (e & 3), ww = w0 + ((e >> 2) & 3), c = e >> 4;
                v[u] = (qin && e >= 0 && hh >= 0 && hh < H && ww >= 0 && ww < W)
                           ? static_cast<float>(img[(static_cast<int64_t>(hh) * W + ww) * Ci + c])
                           : 0.0f;
            }
            bx[ks] = M::pack(v);
        }
        for (int ob = 0; ob < nmt; ob += OT) {
            floatx4 acc[OT];
#pragma unroll
            for (int mt = 0; mt < OT; ++mt) {
                const int o0 = (ob + mt) * 16 + 4 * g;
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[mt][v] = (o0 + v < O) ? b[o0 + v] : 0.0f;
            }
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
                for (int mt = 0; mt < OT; ++mt) {
                    const int o = (ob + mt) * 16 + r;
                    const Frag a = (o < O) ? *reinterpret_cast<const Frag *>(ws + o * KP + ks * 32 + 8 * g)
                                           : M::zero();
                    acc[mt] = M::run(a, bx[ks], acc[mt]);
                }
            }
#pragma unroll
            for (int mt = 0; mt < OT; ++mt) {
                const int o0 = (ob + mt) * 16 + 4 * g;
                if (qin && o0 < O) {  // O is a multiple of 8: all four outputs exist
                    float out[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) out[v] = clamp_act(acc[mt][v], lo, hi);
                    io<T>::store4(y + q * O + o0, out);
                }
            }
        }
    }
}

}  // namespace dynconv
