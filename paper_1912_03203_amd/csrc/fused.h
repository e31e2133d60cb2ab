// fused.h -- one-launch gated block for image widths up to 64 (gfx950).
//
// k_block_fused runs a whole spatially gated inverted-residual block
// (Sec. 3.2) for one band of R image rows per workgroup, keeping every
// intermediate on chip:
//   1. the band's hard-mask rows (and one row above and below) become 64-bit
//      ballot words; the active set A and its 3x3 dilation D (the positions
//      the expansion must cover, rows h0-1 .. h0+R) are compacted in raster
//      order into LDS lists with popcount ranks;
//   2. x of the band's region rows (h0-1 .. h0+R) is copied into LDS at
//      kernel start, one contiguous stretch of NHWC (the expansion's B
//      operand; the band's own rows later become the output tile);
//   3. for each 32-channel slice of the hidden layer (the slice's weights
//      staged in LDS, the next slice's loads in flight meanwhile):
//      expansion of the rows of D (MFMA, bias as the accumulator's start) +
//      activation, stored at the row's position in a zero-bordered
//      (R+2) x (W+2) region array, so that the depthwise 3x3 at an active
//      position reads its 9 taps at fixed offsets from its own row (taps
//      outside the image land on the zero border; taps inside it are in D);
//      the depthwise output (fp32 sums, taps in registers, activation) is
//      the B operand of the projection (MFMA), accumulated over the slices;
//   4. epilogue: y = x + F at the active positions of the band's own rows in
//      LDS (inactive positions keep x bit for bit), one coalesced store of
//      the band, and the next block's mask unit on the stored values (the
//      fp32 fused multiply-add chain of k_mask).
// The arithmetic of every output element is the one of the kernel chain
// (k_expand, k_dw_project): same operand fragments, same summation order.
// Input and output must be different buffers: neighbouring bands read the
// rows next to this band as their halo.  Band i writes its active and
// dilated counts to band_counts[2i], [2i+1]; k_band_counts sums them.
#pragma once

#include "kernels.h"

namespace dynconv {

constexpr int kFusedMaxRegionRows = 64;     // R + 2
constexpr int kChunk = 32;                  // hidden channels per slice
constexpr int kChunkPad = kChunk + 8;       // padded LDS row of a slice
constexpr int kMaxFusedC = 64;

// Band geometry for at most MAXPOS active positions per band (R*W <= MAXPOS):
// rows of the band, at most 62 (the region of rows h0-1 .. h0+R fits 64).
__host__ __device__ constexpr int fused_rows(int maxpos, int W, int H) {
    int r = maxpos / W;
    if (r > kFusedMaxRegionRows - 2) r = kFusedMaxRegionRows - 2;
    if (r > H) r = H;
    return r < 1 ? 1 : r;
}
// largest zero-bordered region (R+2) x (W+2) over the widths 1..64
__host__ __device__ constexpr int fused_max_region(int maxpos) {
    int m = 0;
    for (int w = 1; w <= kWave; ++w) {
        const int r = fused_rows(maxpos, w, 1 << 20);
        if ((r + 2) * (w + 2) > m) m = (r + 2) * (w + 2);
    }
    return m;
}

template <int MAXPOS, int NW>
struct BandShape {
    static constexpr int kThreads = NW * kWave;                // workgroup size
    static constexpr int kMaxNeed = MAXPOS + 2 * kWave;       // region positions (R+2)*W
    static constexpr int kMaxRegion = fused_max_region(MAXPOS);
    static constexpr int kNeedTiles = (kMaxNeed / 16 + NW - 1) / NW;   // 16-row tiles per wave
    static constexpr int kActTiles = (MAXPOS / 16 + NW - 1) / NW;
};

// Weights of one 32-channel slice of the hidden layer.
template <typename T, int MAXC>
struct SliceWeights {
    alignas(16) T w1[kChunk][MAXC + 8];    // expansion rows e (slice-local), c fastest, padded
    alignas(16) T w3[MAXC][kChunkPad];     // projection rows c, slice channels fastest
    alignas(16) T w2[9][kChunk];           // depthwise taps, transposed
    alignas(16) float b1[kChunk];
    alignas(16) float b2[kChunk];
};

template <typename T, int MAXC, int MAXPOS>
struct FusedLds {
    typedef BandShape<MAXPOS, 1> B;
    uint64_t nw[kFusedMaxRegionRows];   // dilated positions (of the band's actives) per region row
    uint64_t aw[kFusedMaxRegionRows];   // active positions (own rows only)
    uint64_t gw[kFusedMaxRegionRows];   // mask words of region rows (image rows h0-1+rr)
    int need_off[kFusedMaxRegionRows + 1];
    int act_off[kFusedMaxRegionRows + 1];
    int16_t need[B::kMaxNeed];          // zero-bordered region index rr*(W+2) + w+1, raster order
    int16_t act[MAXPOS];
    alignas(16) float b3[MAXC];
    SliceWeights<T, MAXC> wt[2];        // double-buffered slice weights
    alignas(16) T xs[B::kMaxNeed][MAXC + 8];  // x of the region rows (rr*W + w), padded rows;
                                              // the band's own rows become y
    alignas(16) T h1r[B::kMaxRegion][kChunkPad];  // the slice, zero-bordered region layout
};

// Cooperative global -> register -> LDS staging of one slice's weights: each
// thread owns kStageSlots 16-byte pieces (zero beyond E).
template <typename T, int MAXC, int NT>
struct SliceStager {
    static constexpr int kPer16 = 16 / static_cast<int>(sizeof(T));
    static constexpr int kPieces = 2 * kChunk * MAXC / kPer16 + kChunk * 9 / kPer16 + 2 * kChunk / 4;
    static constexpr int kStageSlots = (kPieces + NT - 1) / NT;
    uint4 v[kStageSlots];
    // piece index p enumerates, in order: w1 rows (32 x C), w3 rows (C x 32),
    // w2 (32 channels x 9 taps, read as [e][9]), b1, b2
    __device__ __forceinline__ void load(const T *w1, const T *w2, const T *w3, const float *b1,
                                         const float *b2, int C, int E, int ec, int tid) {
        constexpr int per16 = kPer16;
        const int n1 = kChunk * C / per16, n3 = C * kChunk / per16;
        const int e_base = ec * kChunk;
#pragma unroll
        for (int sl = 0; sl < kStageSlots; ++sl) {
            const int p = tid + sl * NT;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (p < n1) {
                const int e = p / (C / per16), c = (p % (C / per16)) * per16;
                if (e_base + e < E)
                    val = *reinterpret_cast<const uint4 *>(w1 + static_cast<int64_t>(e_base + e) * C + c);
            } else if (p < n1 + n3) {
                const int q = p - n1;
                const int c = q / (kChunk / per16), e = (q % (kChunk / per16)) * per16;
                if (e_base + e < E)
                    val = *reinterpret_cast<const uint4 *>(w3 + static_cast<int64_t>(c) * E + e_base + e);
            } else if (p < n1 + n3 + kChunk * 9 / per16) {
                // w2 [E][9] for the slice's 32 channels is 288 contiguous elements;
                // E - e_base is a multiple of 16, so no piece straddles E
                const int q = p - n1 - n3;
                const int first = q * per16;
                if (first / 9 < E - e_base)
                    val = *reinterpret_cast<const uint4 *>(w2 + static_cast<int64_t>(e_base) * 9 + first);
            } else if (p < n1 + n3 + kChunk * 9 / per16 + 2 * kChunk / 4) {
                const int q = p - n1 - n3 - kChunk * 9 / per16;
                const float *b = (q < kChunk / 4) ? b1 : b2;
                const int e = (q % (kChunk / 4)) * 4;
                if (e_base + e < E) val = *reinterpret_cast<const uint4 *>(b + e_base + e);
            }
            v[sl] = val;
        }
    }
    __device__ __forceinline__ void store(SliceWeights<T, MAXC> &dst, int C, int E, int ec,
                                          int tid) const {
        constexpr int per16 = kPer16;
        const int n1 = kChunk * C / per16, n3 = C * kChunk / per16;
        const int e_lim = E - ec * kChunk;
#pragma unroll
        for (int sl = 0; sl < kStageSlots; ++sl) {
            const int p = tid + sl * NT;
            if (p < n1) {
                const int e = p / (C / per16), c = (p % (C / per16)) * per16;
                *reinterpret_cast<uint4 *>(&dst.w1[e][c]) = v[sl];
            } else if (p < n1 + n3) {
                const int q = p - n1;
                const int c = q / (kChunk / per16), e = (q % (kChunk / per16)) * per16;
                *reinterpret_cast<uint4 *>(&dst.w3[c][e]) = v[sl];
            } else if (p < n1 + n3 + kChunk * 9 / per16) {
                const int q = p - n1 - n3;
                const T *vals = reinterpret_cast<const T *>(&v[sl]);
#pragma unroll
                for (int u = 0; u < per16; ++u) {
                    const int idx = q * per16 + u;  // = e * 9 + k
                    const int e = idx / 9, k = idx % 9;
                    dst.w2[k][e] = (e < e_lim) ? vals[u] : static_cast<T>(0.0f);
                }
            } else if (p < n1 + n3 + kChunk * 9 / per16 + 2 * kChunk / 4) {
                const int q = p - n1 - n3 - kChunk * 9 / per16;
                float *b = (q < kChunk / 4) ? dst.b1 : dst.b2;
                *reinterpret_cast<uint4 *>(&b[(q % (kChunk / 4)) * 4]) = v[sl];
            }
        }
    }
};

template <typename T, bool DENSE, int MAXKS, int MAXMT, int MAXC, int MAXPOS, int NW, int WPE>
__global__ void __launch_bounds__(NW * kWave) __attribute__((amdgpu_waves_per_eu(WPE)))
k_block_fused(const T *__restrict__ xin, T *__restrict__ yout, int N, int H, int W, int C, int E,
              int R, const uint8_t *__restrict__ mask_in,
              const T *__restrict__ w1, const float *__restrict__ b1, int act1,
              const T *__restrict__ w2, const float *__restrict__ b2, int act2,
              const T *__restrict__ w3, const float *__restrict__ b3, int act3,
              const float *__restrict__ wm_next, float bm_next, uint8_t *__restrict__ mask_next,
              int32_t *__restrict__ band_counts) {
    typedef mma<T> M;
    typedef BandShape<MAXPOS, NW> BS;
    constexpr int kNeedTiles = BS::kNeedTiles, kActTiles = BS::kActTiles;
    constexpr int NT = BS::kThreads;
    __shared__ FusedLds<T, MAXC, MAXPOS> L;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int r = lane % 16, g = lane / 16;

    // Band index, XCD-aware: workgroup i runs on XCD i % 8, so consecutive
    // bands (which share halo rows) go to the same XCD.
    const int nbh = (H + R - 1) / R;
    const int nbands = N * nbh;
    const int per_xcd = (nbands + 7) / 8;
    const int band = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (band >= nbands) return;  // uniform per workgroup
    const int n = band / nbh;
    const int h0 = (band % nbh) * R;
    const int rows_out = min(R, H - h0);
    const int nreg = rows_out + 2;
    const int WP = W + 2;  // zero-bordered region row length
    const uint64_t full = (W == 64) ? ~0ull : ((1ull << W) - 1ull);
    const int64_t img = static_cast<int64_t>(n) * H;
    const int nchunks = (E + kChunk - 1) / kChunk;
    const float lo1 = act_lo(act1), hi1 = act_hi(act1);
    const float lo2 = act_lo(act2), hi2 = act_hi(act2);
    const float lo3 = act_lo(act3), hi3 = act_hi(act3);
    constexpr int per16 = 16 / static_cast<int>(sizeof(T));

    // All of these only depend on the arguments, so their loads overlap:
    // the first slice's weights, the projection bias, and x of every region
    // row inside the image (rows h0-1 .. h0+R: one contiguous NHWC stretch).
    SliceStager<T, MAXC, NT> stage;
    stage.load(w1, w2, w3, b1, b2, C, E, 0, tid);
    for (int c = tid; c < C; c += NT) L.b3[c] = b3[c];
    {
        const int r_first = (h0 == 0) ? 1 : 0;          // region row of image row max(h0-1, 0)
        const int r_last = (h0 + rows_out < H) ? nreg - 1 : nreg - 2;
        const int vpr = C / per16;                      // 16-byte pieces per position
        const int nvec = (r_last - r_first + 1) * W * vpr;
        const uint4 *src = reinterpret_cast<const uint4 *>(xin + (img + h0 - 1 + r_first) * W * C);
        for (int i = tid; i < nvec; i += NT)
            *reinterpret_cast<uint4 *>(&L.xs[r_first * W + i / vpr][(i % vpr) * per16]) = src[i];
    }
    {   // zero region: its border and out-of-image rows are never written again
        uint4 *z = reinterpret_cast<uint4 *>(&L.h1r[0][0]);
        constexpr int nz = BS::kMaxRegion * kChunkPad * static_cast<int>(sizeof(T)) / 16;
        for (int i = tid; i < nz; i += NT) z[i] = make_uint4(0, 0, 0, 0);
    }

    // ---- 1. mask words, dilation, lists
    for (int rr = wave; rr < nreg; rr += NW) {
        const int hh = h0 - 1 + rr;
        bool bit = false;
        if (hh >= 0 && hh < H && lane < W)
            bit = DENSE ? true : mask_in[(img + hh) * W + lane] != 0;
        const uint64_t b = __ballot(bit);
        if (lane == 0) L.gw[rr] = b;
    }
    __syncthreads();
    if (wave == 0) {
        // lane rr computes region row rr (nreg <= 64)
        const int rr = lane;
        uint64_t a = 0, nwd = 0, dil_own = 0;
        if (rr < nreg) {
            const bool own = rr >= 1 && rr <= rows_out;
            const int hh = h0 - 1 + rr;
            const bool inimg = hh >= 0 && hh < H;
            const uint64_t above = (rr - 1 >= 1 && rr - 1 <= rows_out) ? L.gw[rr - 1] : 0ull;
            const uint64_t below = (rr + 1 >= 1 && rr + 1 <= rows_out) ? L.gw[rr + 1] : 0ull;
            a = own ? L.gw[rr] : 0ull;
            const uint64_t v = above | a | below;
            nwd = inimg ? ((v | (v << 1) | (v >> 1)) & full) : 0ull;
            if (own) {
                const uint64_t gv = L.gw[rr - 1] | L.gw[rr] | L.gw[rr + 1];
                dil_own = (gv | (gv << 1) | (gv >> 1)) & full;
            }
            L.aw[rr] = a;
            L.nw[rr] = nwd;
        }
        // inclusive scans of the per-row counts across the wave
        const int cn = __popcll(nwd), ca = __popcll(a);
        int sn = cn, sa = ca;
        for (int off = 1; off < kWave; off <<= 1) {
            const int tn = __shfl_up(sn, off), ta = __shfl_up(sa, off);
            if (lane >= off) {
                sn += tn;
                sa += ta;
            }
        }
        if (rr < nreg) {
            L.need_off[rr] = sn - cn;
            L.act_off[rr] = sa - ca;
        }
        if (rr == nreg - 1) {
            L.need_off[nreg] = sn;
            L.act_off[nreg] = sa;
        }
        if (!DENSE && band_counts) {
            // this band's active and dilated counts (a plain store per band:
            // atomics on one address from every XCD serialise)
            int pa = ca, pd = __popcll(dil_own);
            for (int off = 32; off > 0; off >>= 1) {
                pa += __shfl_down(pa, off);
                pd += __shfl_down(pd, off);
            }
            if (lane == 0) *reinterpret_cast<int2 *>(band_counts + 2 * band) = make_int2(pa, pd);
        }
    }
    __syncthreads();
    const uint64_t lt = lanemask_lt(lane);
    for (int rr = wave; rr < nreg; rr += NW) {
        if (lane < W) {
            const uint64_t nwd = L.nw[rr], awd = L.aw[rr];
            const int16_t q = static_cast<int16_t>(rr * WP + lane + 1);
            if ((nwd >> lane) & 1ull) L.need[L.need_off[rr] + __popcll(nwd & lt)] = q;
            if ((awd >> lane) & 1ull) L.act[L.act_off[rr] + __popcll(awd & lt)] = q;
        }
    }
    stage.store(L.wt[0], C, E, 0, tid);
    __syncthreads();
    const int n_need = L.need_off[nreg];
    const int n_act = L.act_off[nreg];
    T (*yrows)[MAXC + 8] = &L.xs[W];  // the band's own rows (region rows 1..rows_out)

    if (n_act > 0) {
        // region rows of this wave's need and active tiles: index into the
        // zero-bordered region (h1r) and into the unbordered x rows (xs)
        int nq[kNeedTiles], nx[kNeedTiles];
#pragma unroll
        for (int j = 0; j < kNeedTiles; ++j) {
            const int i = (wave + NW * j) * 16 + r;
            const int q = (i < n_need) ? static_cast<int>(L.need[i]) : -1;
            nq[j] = q;
            nx[j] = (q >= 0) ? (q / WP) * W + q % WP - 1 : W;  // past n_need: any row, never stored
        }
        int aq[kActTiles];
#pragma unroll
        for (int j = 0; j < kActTiles; ++j) {
            const int i = (wave + NW * j) * 16 + r;
            aq[j] = (i < n_act) ? static_cast<int>(L.act[i]) : -1;
        }
        floatx4 acc[kActTiles][MAXMT];
#pragma unroll
        for (int j = 0; j < kActTiles; ++j)
#pragma unroll
            for (int mt = 0; mt < MAXMT; ++mt) {
                const int c0 = mt * 16 + 4 * g;
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[j][mt][v] = (c0 < C) ? L.b3[c0 + v] : 0.0f;
            }
        const int row_bytes = WP * kChunkPad * static_cast<int>(sizeof(T));
        constexpr int col_bytes = kChunkPad * static_cast<int>(sizeof(T));

        for (int ec = 0; ec < nchunks; ++ec) {
            const SliceWeights<T, MAXC> &sw = L.wt[ec & 1];
            if (ec + 1 < nchunks) stage.load(w1, w2, w3, b1, b2, C, E, ec + 1, tid);
            // ---- 3a. expansion of this slice into the region array
            typename M::frag a1[2][MAXKS];
            floatx4 binit[2];
#pragma unroll
            for (int m = 0; m < 2; ++m) {
#pragma unroll
                for (int ks = 0; ks < MAXKS; ++ks) {
                    const int c0 = ks * 32 + g * 8;
                    a1[m][ks] = (c0 < C) ? M::load(&sw.w1[m * 16 + r][c0]) : M::zero();
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) binit[m][v] = sw.b1[m * 16 + 4 * g + v];
            }
#pragma unroll
            for (int j = 0; j < kNeedTiles; ++j) {
                const int t = wave + NW * j;
                if (t * 16 < n_need) {
                    typename M::frag bxs[MAXKS];
#pragma unroll
                    for (int ks = 0; ks < MAXKS; ++ks) {
                        const int c0 = ks * 32 + g * 8;
                        bxs[ks] = (c0 < C) ? M::load(&L.xs[nx[j]][c0]) : M::zero();
                    }
#pragma unroll
                    for (int m = 0; m < 2; ++m) {
                        floatx4 d = binit[m];
#pragma unroll
                        for (int ks = 0; ks < MAXKS; ++ks) d = M::run(a1[m][ks], bxs[ks], d);
                        const int e0 = ec * kChunk + m * 16 + 4 * g;
                        if (nq[j] >= 0 && e0 < E) {
                            float o[4];
#pragma unroll
                            for (int v = 0; v < 4; ++v) o[v] = clamp_act(d[v], lo1, hi1);
                            io<T>::store4(&L.h1r[nq[j]][m * 16 + 4 * g], o);
                        }
                    }
                }
            }
            if (ec + 1 < nchunks) stage.store(L.wt[(ec + 1) & 1], C, E, ec + 1, tid);
            __syncthreads();
            // ---- 3b. depthwise at the active positions + projection slice
            const int e8 = ec * kChunk + 8 * g;
            const bool ein = e8 < E;
            typename io<T>::vec8 wk[9];  // the lane's 8 channels of each tap, packed
#pragma unroll
            for (int k = 0; k < 9; ++k) wk[k] = io<T>::raw8(&sw.w2[k][8 * g]);
            float bk[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) bk[u] = sw.b2[8 * g + u];
            typename M::frag a3[MAXMT];
#pragma unroll
            for (int mt = 0; mt < MAXMT; ++mt) {
                const int c = mt * 16 + r;
                a3[mt] = (ein && c < C) ? M::load(&sw.w3[c][8 * g]) : M::zero();
            }
            const char *h1base = reinterpret_cast<const char *>(&L.h1r[0][8 * g]);
#pragma unroll
            for (int j = 0; j < kActTiles; ++j) {
                const int t = wave + NW * j;
                if (t * 16 < n_act) {
                    float hv[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) hv[u] = 0.0f;
                    if (aq[j] >= 0 && ein) {
                        const char *own = h1base + aq[j] * col_bytes;
                        float s[8];
#pragma unroll
                        for (int u = 0; u < 8; ++u) s[u] = bk[u];
#pragma unroll
                        for (int k = 0; k < 9; ++k) {
                            const int off = (k / 3 - 1) * row_bytes + (k % 3 - 1) * col_bytes;
                            float v[8];
                            io<T>::load8(reinterpret_cast<const T *>(own + off), v);
#pragma unroll
                            for (int u = 0; u < 8; ++u)
                                s[u] = __builtin_fmaf(static_cast<float>(wk[k][u]), v[u], s[u]);
                        }
#pragma unroll
                        for (int u = 0; u < 8; ++u) hv[u] = clamp_act(s[u], lo2, hi2);
                    }
                    const typename M::frag bf = M::pack(hv);
#pragma unroll
                    for (int mt = 0; mt < MAXMT; ++mt) acc[j][mt] = M::run(a3[mt], bf, acc[j][mt]);
                }
            }
            __syncthreads();
        }
        // ---- 4a. residual sum at the active positions, in the band's own x rows
#pragma unroll
        for (int j = 0; j < kActTiles; ++j) {
            if (aq[j] >= 0) {
                const int q = (aq[j] / WP - 1) * W + aq[j] % WP - 1;  // own-row index
#pragma unroll
                for (int mt = 0; mt < MAXMT; ++mt) {
                    const int c0 = mt * 16 + 4 * g;
                    if (c0 < C) {
                        float xv[4], o[4];
                        io<T>::load4(&yrows[q][c0], xv);
#pragma unroll
                        for (int v = 0; v < 4; ++v) o[v] = xv[v] + clamp_act(acc[j][mt][v], lo3, hi3);
                        io<T>::store4(&yrows[q][c0], o);
                    }
                }
            }
        }
        __syncthreads();
    }
    // ---- 4b. store the band (inactive positions: x unchanged)
    {
        const int vpr = C / per16;
        const int nvec = rows_out * W * vpr;
        uint4 *dst = reinterpret_cast<uint4 *>(yout + (img + h0) * W * C);
        for (int i = tid; i < nvec; i += NT)
            dst[i] = *reinterpret_cast<const uint4 *>(&yrows[i / vpr][(i % vpr) * per16]);
    }
    // ---- 4c. the next block's mask unit on the stored values
    if (mask_next) {
        for (int q = tid; q < rows_out * W; q += NT) {
            const T *row = &yrows[q][0];
            float a = 0.0f;
            for (int c0 = 0; c0 < C; c0 += 8) {
                float v[8];
                io<T>::load8(row + c0, v);
#pragma unroll
                for (int u = 0; u < 8; ++u) a = __builtin_fmaf(wm_next[c0 + u], v[u], a);
            }
            const float m = a + bm_next;
            mask_next[(img + h0) * W + q] = (m > 0.0f) ? 1 : 0;
        }
    }
}

// counts[2b], counts[2b+1] = sums of the per-band counts of block b
// (one workgroup per block, fixed summation order).
__global__ void __launch_bounds__(kBlock)
k_band_counts(const int32_t *__restrict__ band_counts, int nbands, int32_t *__restrict__ counts) {
    __shared__ int2 part[kBlock];
    const int b = blockIdx.x;
    const int2 *src = reinterpret_cast<const int2 *>(band_counts) + static_cast<int64_t>(b) * nbands;
    int2 acc = make_int2(0, 0);
    for (int i = threadIdx.x; i < nbands; i += kBlock) {
        const int2 v = src[i];
        acc.x += v.x;
        acc.y += v.y;
    }
    part[threadIdx.x] = acc;
    __syncthreads();
    for (int off = kBlock / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) {
            part[threadIdx.x].x += part[threadIdx.x + off].x;
            part[threadIdx.x].y += part[threadIdx.x + off].y;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        counts[2 * b] = part[0].x;
        counts[2 * b + 1] = part[0].y;
    }
}

}  // namespace dynconv
