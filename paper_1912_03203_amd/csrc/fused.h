// fused.h -- one-launch gated block (gfx950).
//
// k_block_fused runs a whole spatially gated inverted-residual block
// (Sec. 3.2) for one patch of R image rows x Wu columns per workgroup,
// keeping every intermediate on chip:
//   1. the hard-mask rows of the patch's region (the patch plus a one-pixel
//      ring: rows h0-1 .. h0+R, columns w0-1 .. w0+Wu) become 64-bit ballot
//      words; the patch's active set A and the part of its 3x3 dilation the
//      expansion must cover (every in-image region position next to an
//      active one) are compacted in raster order into LDS lists with
//      popcount ranks;
//   2. x at every in-image region position is copied into LDS; each wave
//      keeps the expansion's B fragments of its needed positions in
//      registers for all slices; the patch's own positions become the output;
//   3. for each 32-channel slice of the hidden layer: expansion of the
//      needed positions (MFMA, bias as the accumulator's start) +
//      activation, stored at the position's slot of a (R+2) x (Wu+2) region
//      array, so that the depthwise 3x3 at an active position reads its 9
//      taps at fixed offsets (slots outside the image stay zero, slots inside
//      it were expanded); the depthwise output (fp32 sums, activation) is the
//      B operand of the projection (MFMA), accumulated over the slices.  The
//      expansion weights and the depthwise/projection weights of a slice sit
//      in one LDS buffer each: the next slice's expansion weights are written
//      while the depthwise runs, its depthwise/projection weights while the
//      next expansion runs, each loaded from memory one slice ahead;
//   4. epilogue: y = x + F at the active positions (inactive positions keep
//      x bit for bit), a coalesced store of the patch, and the next block's
//      mask unit on the stored values (the fp32 multiply-add chain of k_mask).
// Patches are small (at most 256 positions) and many, so the hardware
// dispatcher spreads patches of very different active counts over the CUs.
// The arithmetic of every output element is the one of the kernel chain
// (k_expand, k_dw_project): same operand fragments, same summation order.
// Input and output must be different buffers: neighbouring patches read the
// positions next to this one as their ring.  Patch i writes its active and
// dilated counts to band_counts[2i], [2i+1]; k_band_counts sums them.
// The first block of a stack may compute its own mask (wm_self) from the
// staged x instead of reading one.  mask_mode selects the hard decision
// (mask_decision: G-Binary or G-Softmax).
#pragma once

#include "kernels.h"

#include <type_traits>

namespace dynconv {

constexpr int kChunk = 32;                  // hidden channels per slice
constexpr int kChunkPad = kChunk + 8;       // padded LDS row of a slice
constexpr int kMaxFusedC = 64;    // fp32
constexpr int kMaxFusedC16 = 128; // fp16 / bf16
constexpr int kPatchMaxCols = 32;           // Wu
constexpr int kPatchMaxRows = 50;           // R

// A patch configuration: at most OWN own positions and REGION region slots
// per patch, NW waves per workgroup, register budget for WPE waves per SIMD.
template <int OWN, int REGION, int NW, int WPE>
struct PatchCfg {
    static constexpr int kOwn = OWN, kRegion = REGION, kWaves = NW, kWpe = WPE;
    static constexpr int kThreads = NW * kWave;
};
// Per element type and channel bound, the largest patches whose LDS lets the
// most waves run per CU:
//   16-bit, C <= 32: 8 x 32 patches, 8 waves, two workgroups per CU
//   16-bit, C <= 64: 4 x 32 patches, 4 waves, two workgroups per CU
//   fp32,   C <= 32: 8 x 32 patches, 8 waves, one workgroup per CU
//   fp32,   C <= 64: 4 x 32 patches, 4 waves, one workgroup per CU
//   16-bit, C <= 128: 64-position patches, 4 waves, two workgroups per CU
template <typename T, int MAXC> struct PatchCfgOf;
template <int MAXC> struct PatchCfgOf<float, MAXC> {
    typedef typename std::conditional<MAXC <= 32, PatchCfg<256, 340, 8, 2>, PatchCfg<128, 208, 4, 1>>::type type;
};
template <int MAXC> struct PatchCfgOf<half_t, MAXC> {
    typedef typename std::conditional<
        MAXC <= 32, PatchCfg<256, 340, 8, 4>,
        typename std::conditional<MAXC <= 64, PatchCfg<128, 208, 4, 2>, PatchCfg<64, 108, 4, 2>>::type>::type type;
};
template <int MAXC> struct PatchCfgOf<bf16_t, MAXC> : PatchCfgOf<half_t, MAXC> {};

// Patch geometry: the image width is cut into equal column strips of at most
// 32, the height into strips of R rows, with R * Wu <= own and the region
// (R+2) x (Wu+2) <= region.  Small images get shorter row strips until the
// batch has at least kMinPatches patches, so that the launch still covers
// the chip.
constexpr int kMinPatches = 256;
struct PatchGeom {
    int R, Wu, nph, npw;
};
__host__ __device__ inline PatchGeom patch_geom(int N, int H, int W, int own, int region) {
    PatchGeom p;
    const int strips = (W + kPatchMaxCols - 1) / kPatchMaxCols;
    p.Wu = (W + strips - 1) / strips;
    p.npw = (W + p.Wu - 1) / p.Wu;
    int r = own / p.Wu;
    const int rr = region / (p.Wu + 2) - 2;
    if (r > rr) r = rr;
    if (r > kPatchMaxRows) r = kPatchMaxRows;
    if (r > H) r = H;
    while (r > 1 && static_cast<int64_t>(N) * ((H + r - 1) / r) * p.npw < kMinPatches) --r;
    p.R = r < 1 ? 1 : r;
    p.nph = (H + p.R - 1) / p.R;
    return p;
}

// Weights of one 32-channel slice of the hidden layer, in the two parts that
// different phases of the slice read.
template <typename T, int MAXC>
struct ExpandWeights {
    alignas(16) T w1[kChunk][MAXC + 8];    // expansion rows e (slice-local), c fastest, padded
    alignas(16) float b1[kChunk];
};
template <typename T, int MAXC>
struct DwProjWeights {
    alignas(16) T w3[MAXC][kChunkPad];     // projection rows c, slice channels fastest
    alignas(16) T w2[9][kChunk];           // depthwise taps, transposed
    alignas(16) float b2[kChunk];
};

template <typename T, int MAXC, class CFG, bool SHUF = false>
struct PatchLds {
    static constexpr int kRows = kPatchMaxRows + 2;
    uint64_t nw[kRows];                 // needed slots per region row (bit = region column)
    uint64_t aw[kRows];                 // active own positions per region row
    uint64_t gw[kRows];                 // mask words of the region rows
    int need_off[kRows + 1];
    int act_off[kRows + 1];
    int16_t need[CFG::kRegion];         // region slot rr*(cols+2) + c, raster order
    int16_t act[CFG::kOwn];
    alignas(16) float b3[MAXC];
    ExpandWeights<T, MAXC> we;
    DwProjWeights<T, MAXC> wd;
    alignas(16) T xs[CFG::kRegion][MAXC + 8];       // x at region slots; own slots become y
    alignas(16) T h1r[CFG::kRegion + 1][kChunkPad]; // the slice in region layout + a spare row
    // ShuffleNetV2 rows: the pass-through half of the own positions
    alignas(16) T x1s[SHUF ? CFG::kOwn : 1][SHUF ? MAXC : 1];
};

// Inclusive prefix sum over the 64 lanes of a wave with DPP row operations:
// shifts by 1, 2, 4, 8 within each row of 16 lanes, then lane 15 of rows 0
// and 2 added into rows 1 and 3, then lane 31 into rows 2 and 3.
__device__ __forceinline__ int wave_scan_incl(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
    return v;
}

// Cooperative global -> register -> LDS staging of one part of a slice's
// weights: each thread owns kSlots 16-byte pieces (zero beyond E).
template <typename T, int MAXC, int NT>
struct ExpandStager {
    static constexpr int kPer16 = 16 / static_cast<int>(sizeof(T));
    static constexpr int kPieces = kChunk * MAXC / kPer16 + kChunk / 4;
    static constexpr int kSlots = (kPieces + NT - 1) / NT;
    uint4 v[kSlots];
    // pieces: w1 rows (32 x C), then b1
    __device__ __forceinline__ void load(const T *w1, const float *b1, int C, int E, int ec, int tid) {
        const int n1 = kChunk * C / kPer16;
        const int e_base = ec * kChunk;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            const int p = tid + sl * NT;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (p < n1) {
                const int e = p / (C / kPer16), c = (p % (C / kPer16)) * kPer16;
                if (e_base + e < E)
                    val = *reinterpret_cast<const uint4 *>(w1 + static_cast<int64_t>(e_base + e) * C + c);
            } else if (p < n1 + kChunk / 4) {
                const int e = (p - n1) * 4;
                if (e_base + e < E) val = *reinterpret_cast<const uint4 *>(b1 + e_base + e);
            }
            v[sl] = val;
        }
    }
    __device__ __forceinline__ void store(ExpandWeights<T, MAXC> &dst, int C, int tid) const {
        const int n1 = kChunk * C / kPer16;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            const int p = tid + sl * NT;
            if (p < n1) {
                const int e = p / (C / kPer16), c = (p % (C / kPer16)) * kPer16;
                *reinterpret_cast<uint4 *>(&dst.w1[e][c]) = v[sl];
            } else if (p < n1 + kChunk / 4) {
                *reinterpret_cast<uint4 *>(&dst.b1[(p - n1) * 4]) = v[sl];
            }
        }
    }
};

template <typename T, int MAXC, int NT>
struct DwProjStager {
    static constexpr int kPer16 = 16 / static_cast<int>(sizeof(T));
    static constexpr int kPieces = MAXC * kChunk / kPer16 + kChunk / 4;
    static constexpr int kSlots = (kPieces + NT - 1) / NT;
    static constexpr int kTaps = kChunk * 9;                 // depthwise weights of a slice
    static constexpr int kTapSlots = (kTaps + NT - 1) / NT;
    uint4 v[kSlots];
    T t[kTapSlots];
    // 16-byte pieces: w3 rows (C x 32), then b2.  Depthwise weights: one
    // element per thread (slice element j = 9 e + k of w2 [E][9]), stored
    // transposed as w2[k][e]: a load and a 2-byte store per thread, so no
    // thread packs values whose loads are still in flight.
    __device__ __forceinline__ void load(const T *w2, const T *w3, const float *b2, int C, int E, int ec,
                                         int tid) {
        const int n3 = C * kChunk / kPer16;
        const int e_base = ec * kChunk;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            const int p = tid + sl * NT;
            uint4 val = make_uint4(0, 0, 0, 0);
            if (p < n3) {
                const int c = p / (kChunk / kPer16), e = (p % (kChunk / kPer16)) * kPer16;
                if (e_base + e < E)
                    val = *reinterpret_cast<const uint4 *>(w3 + static_cast<int64_t>(c) * E + e_base + e);
            } else if (p < n3 + kChunk / 4) {
                const int e = (p - n3) * 4;
                if (e_base + e < E) val = *reinterpret_cast<const uint4 *>(b2 + e_base + e);
            }
            v[sl] = val;
        }
#pragma unroll
        for (int sl = 0; sl < kTapSlots; ++sl) {
            const int j = tid + sl * NT;
            t[sl] = static_cast<T>(0.0f);
            if (j < kTaps && e_base + j / 9 < E) t[sl] = w2[static_cast<int64_t>(e_base) * 9 + j];
        }
    }
    __device__ __forceinline__ void store(DwProjWeights<T, MAXC> &dst, int C, int tid) const {
        const int n3 = C * kChunk / kPer16;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            const int p = tid + sl * NT;
            if (p < n3) {
                const int c = p / (kChunk / kPer16), e = (p % (kChunk / kPer16)) * kPer16;
                *reinterpret_cast<uint4 *>(&dst.w3[c][e]) = v[sl];
            } else if (p < n3 + kChunk / 4) {
                *reinterpret_cast<uint4 *>(&dst.b2[(p - n3) * 4]) = v[sl];
            }
        }
#pragma unroll
        for (int sl = 0; sl < kTapSlots; ++sl) {
            const int j = tid + sl * NT;
            if (j < kTaps) dst.w2[j % 9][j / 9] = t[sl];
        }
    }
};

template <typename T, bool DENSE, int MAXKS, int MAXMT, int MAXC, class CFG, bool SHUF>
__global__ void __launch_bounds__(CFG::kThreads) __attribute__((amdgpu_waves_per_eu(CFG::kWpe)))
k_block_fused(const T *__restrict__ xin, T *__restrict__ yout, int N, int H, int W, int C, int E,
              int R, int Wu, int cb, const uint8_t *__restrict__ mask_in,
              const float *__restrict__ wm_self, float bm_self, uint8_t *__restrict__ mask_self,
              const T *__restrict__ w1, const float *__restrict__ b1, int act1,
              const T *__restrict__ w2, const float *__restrict__ b2, int act2,
              const T *__restrict__ w3, const float *__restrict__ b3, int act3,
              const float *__restrict__ wm_next, float bm_next, uint8_t *__restrict__ mask_next,
              int32_t *__restrict__ band_counts, int mask_mode) {
    typedef mma<T> M;
    constexpr int NW = CFG::kWaves, NT = CFG::kThreads, kRegion = CFG::kRegion;
    constexpr int kNeedTiles = ((kRegion + 15) / 16 + NW - 1) / NW;  // 16-slot tiles per wave
    constexpr int kActTiles = ((CFG::kOwn + 15) / 16 + NW - 1) / NW;
    __shared__ PatchLds<T, MAXC, CFG, SHUF> L;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int r = lane % 16, g = lane / 16;

    const int nph = (H + R - 1) / R, npw = (W + Wu - 1) / Wu;
    const int npatch = N * nph * npw;
    // XCD-aware: workgroup i runs on XCD i % 8, so consecutive patches
    // (which share ring rows and columns) go to the same XCD.
    const int per_xcd = (npatch + 7) / 8;
    const int patch = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (patch >= npatch) return;  // uniform per workgroup
    const int n = patch / (nph * npw);
    const int h0 = ((patch / npw) % nph) * R;
    const int w0 = (patch % npw) * Wu;
    const int rows_out = min(R, H - h0);
    const int cols_out = min(Wu, W - w0);
    const int nreg = rows_out + 2;
    const int WP = cols_out + 2;  // region row length; region column c is image column w0-1+c
    const int c_lo = (w0 == 0) ? 1 : 0;                      // first in-image region column
    const int c_hi = (w0 + cols_out < W) ? WP : WP - 1;      // one past the last
    const uint64_t img_cols = ((1ull << c_hi) - 1ull) & ~((1ull << c_lo) - 1ull);
    const uint64_t own_cols = ((1ull << (cols_out + 1)) - 1ull) & ~1ull;
    const int64_t img = static_cast<int64_t>(n) * H;
    const int nchunks = (E + kChunk - 1) / kChunk;
    const float lo1 = act_lo(act1), hi1 = act_hi(act1);
    const float lo2 = act_lo(act2), hi2 = act_hi(act2);
    const float lo3 = act_lo(act3), hi3 = act_hi(act3);
    constexpr int per16 = 16 / static_cast<int>(sizeof(T));

    // These only depend on the arguments, so their loads overlap: the first
    // slice's weights, the projection bias, x at the in-image region slots.
    ExpandStager<T, MAXC, NT> stA;
    DwProjStager<T, MAXC, NT> stB;
    stA.load(w1, b1, C, E, 0, tid);
    stB.load(w2, w3, b2, C, E, 0, tid);
    for (int c = tid; c < C; c += NT) L.b3[c] = b3[c];
    // x at the in-image region slots (one 16-byte load in flight per thread:
    // measured faster here than batches of loads, which all patches would
    // issue at once)
    const int r_first = (h0 == 0) ? 1 : 0;
    const int r_last = (h0 + rows_out < H) ? nreg - 1 : nreg - 2;
    const int ncol = c_hi - c_lo;
    if (!SHUF) {
        const int vpr = C / per16;                      // 16-byte pieces per position
        const int per_row = ncol * vpr;
        const int nvec = (r_last - r_first + 1) * per_row;
        for (int i = tid; i < nvec; i += NT) {
            const int rr = r_first + i / per_row, k = i % per_row;
            const int c = c_lo + k / vpr, piece = k % vpr;
            const uint4 *src = reinterpret_cast<const uint4 *>(
                xin + ((img + h0 - 1 + rr) * W + (w0 - 1 + c)) * C);
            *reinterpret_cast<uint4 *>(&L.xs[rr * WP + c][piece * per16]) = src[piece];
        }
    } else {
        // unit rows in 4-byte words, in batches of 8 loads per thread: the
        // second half (the block's input, zero past cb) of every in-image
        // region position into xs, the first half of the own positions into x1s
        constexpr int kB = 8;
        constexpr int wpp = MAXC * static_cast<int>(sizeof(T)) / 4;         // words per staged row
        constexpr int wrow = (MAXC + 8) * static_cast<int>(sizeof(T)) / 4;  // words per xs row
        const int wreal = cb * static_cast<int>(sizeof(T)) / 4;
        const int nvec = (r_last - r_first + 1) * ncol * wpp;
        for (int i0 = tid; i0 < nvec; i0 += kB * NT) {
            uint32_t v2[kB], v1[kB];
            int d2[kB], d1[kB];
#pragma unroll
            for (int k = 0; k < kB; ++k) {
                const int i = i0 + k * NT;
                d2[k] = d1[k] = -1;
                v2[k] = v1[k] = 0u;
                if (i < nvec) {
                    const int pos = i / wpp, wd = i % wpp;
                    const int rr = r_first + pos / ncol, c = c_lo + pos % ncol;
                    const uint32_t *row = reinterpret_cast<const uint32_t *>(
                        xin + ((img + h0 - 1 + rr) * W + (w0 - 1 + c)) * (2 * cb));
                    d2[k] = (rr * WP + c) * wrow + wd;
                    if (wd < wreal) {
                        v2[k] = row[wreal + wd];
                        if (rr >= 1 && rr <= rows_out && c >= 1 && c <= cols_out) {
                            v1[k] = row[wd];
                            d1[k] = ((rr - 1) * cols_out + (c - 1)) * wpp + wd;
                        }
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < kB; ++k) {
                if (d2[k] >= 0) reinterpret_cast<uint32_t *>(&L.xs[0][0])[d2[k]] = v2[k];
                if (d1[k] >= 0) reinterpret_cast<uint32_t *>(&L.x1s[0][0])[d1[k]] = v1[k];
            }
        }
    }
    {   // zero region: slots outside the image are never written again
        uint4 *z = reinterpret_cast<uint4 *>(&L.h1r[0][0]);
        constexpr int nz = kRegion * kChunkPad * static_cast<int>(sizeof(T)) / 16;
        for (int i = tid; i < nz; i += NT) z[i] = make_uint4(0, 0, 0, 0);
    }

    // ---- 1. mask words, dilation, lists
    if (!DENSE && wm_self) __syncthreads();  // the region's x, for the block's own mask unit
    for (int rr = wave; rr < nreg; rr += NW) {
        const int hh = h0 - 1 + rr;
        bool bit = false;
        if (hh >= 0 && hh < H && lane < WP && ((img_cols >> lane) & 1ull)) {
            if (DENSE) {
                bit = true;
            } else if (wm_self) {
                // the mask unit (Eq. 2, Eq. 8 at zero noise) on the staged x: the
                // fp32 multiply-add chain of k_mask, channels ascending from +0,
                // then the bias, strict threshold
                const T *row = &L.xs[rr * WP + lane][0];
                float a = 0.0f;
                for (int c0 = 0; c0 < C; c0 += 8) {
                    float v[8];
                    io<T>::load8(row + c0, v);
#pragma unroll
                    for (int u = 0; u < 8; ++u) a = __builtin_fmaf(wm_self[c0 + u], v[u], a);
                }
                bit = mask_decision(a + bm_self, mask_mode);
                if (mask_self && rr >= 1 && rr <= rows_out && lane >= 1 && lane <= cols_out)
                    mask_self[(img + hh) * W + (w0 - 1 + lane)] = bit ? 1 : 0;
            } else {
                bit = mask_in[(img + hh) * W + (w0 - 1 + lane)] != 0;
            }
        }
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
            const uint64_t above = (rr - 1 >= 1 && rr - 1 <= rows_out) ? (L.gw[rr - 1] & own_cols) : 0ull;
            const uint64_t below = (rr + 1 >= 1 && rr + 1 <= rows_out) ? (L.gw[rr + 1] & own_cols) : 0ull;
            a = own ? (L.gw[rr] & own_cols) : 0ull;
            const uint64_t v = above | a | below;
            nwd = inimg ? ((v | (v << 1) | (v >> 1)) & img_cols) : 0ull;
            if (own) {
                const uint64_t gv = L.gw[rr - 1] | L.gw[rr] | L.gw[rr + 1];
                dil_own = (gv | (gv << 1) | (gv >> 1)) & own_cols;
            }
            L.aw[rr] = a;
            L.nw[rr] = nwd;
        }
        // inclusive scans of the per-row counts across the wave, both counts
        // in one 32-bit value (each total is at most 52 x 64 < 2^16)
        const int cn = __popcll(nwd), ca = __popcll(a);
        const int s2 = wave_scan_incl(cn | (ca << 16));
        const int sn = s2 & 0xffff, sa = s2 >> 16;
        if (rr < nreg) {
            L.need_off[rr] = sn - cn;
            L.act_off[rr] = sa - ca;
        }
        if (rr == nreg - 1) {
            L.need_off[nreg] = sn;
            L.act_off[nreg] = sa;
        }
        if (!DENSE && band_counts) {
            // this patch's active and dilated counts (a plain store per patch:
            // atomics on one address from every XCD serialise)
            const int pa = __builtin_amdgcn_readlane(sa, kWave - 1);
            const int pd = __builtin_amdgcn_readlane(wave_scan_incl(__popcll(dil_own)), kWave - 1);
            if (lane == 0) *reinterpret_cast<int2 *>(band_counts + 2 * patch) = make_int2(pa, pd);
        }
    }
    __syncthreads();
    const uint64_t lt = lanemask_lt(lane);
    for (int rr = wave; rr < nreg; rr += NW) {
        if (lane < WP) {
            const uint64_t nwd = L.nw[rr], awd = L.aw[rr];
            const int16_t q = static_cast<int16_t>(rr * WP + lane);
            if ((nwd >> lane) & 1ull) L.need[L.need_off[rr] + __popcll(nwd & lt)] = q;
            if ((awd >> lane) & 1ull) L.act[L.act_off[rr] + __popcll(awd & lt)] = q;
        }
    }
    stA.store(L.we, C, tid);
    __syncthreads();
    const int n_need = L.need_off[nreg];
    const int n_act = L.act_off[nreg];

    if (n_act > 0) {
        // this wave's needed slots (the expansion's output rows; past n_need:
        // the spare row) and their B fragments, kept for every slice
        int nq[kNeedTiles];
        typename M::frag bx[kNeedTiles][MAXKS];
#pragma unroll
        for (int j = 0; j < kNeedTiles; ++j) {
            const int i = (wave + NW * j) * 16 + r;
            const int q = (i < n_need) ? static_cast<int>(L.need[i]) : -1;
            nq[j] = (q >= 0) ? q : kRegion;
            const int qx = (q >= 0) ? q : WP + 1;  // an own slot; its column is never stored
#pragma unroll
            for (int ks = 0; ks < MAXKS; ++ks) {
                const int c0 = ks * 32 + g * 8;
                bx[j][ks] = (c0 < C) ? M::load(&L.xs[qx][c0]) : M::zero();
            }
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
        if (nchunks > 1) stA.load(w1, b1, C, E, 1, tid);

        for (int ec = 0; ec < nchunks; ++ec) {
            // ---- 3a. expansion of this slice into the region array; meanwhile
            // this slice's depthwise/projection weights go to LDS and the next
            // slice's are requested
            stB.store(L.wd, C, tid);
            if (ec + 1 < nchunks) stB.load(w2, w3, b2, C, E, ec + 1, tid);
            typename M::frag a1[2][MAXKS];
            floatx4 binit[2];
#pragma unroll
            for (int m = 0; m < 2; ++m) {
#pragma unroll
                for (int ks = 0; ks < MAXKS; ++ks) {
                    const int c0 = ks * 32 + g * 8;
                    a1[m][ks] = (c0 < C) ? M::load(&L.we.w1[m * 16 + r][c0]) : M::zero();
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) binit[m][v] = L.we.b1[m * 16 + 4 * g + v];
            }
#pragma unroll
            for (int j = 0; j < kNeedTiles; ++j) {
                const int t = wave + NW * j;
                if (t * 16 < n_need) {
#pragma unroll
                    for (int m = 0; m < 2; ++m) {
                        floatx4 d = binit[m];
#pragma unroll
                        for (int ks = 0; ks < MAXKS; ++ks) d = M::run(a1[m][ks], bx[j][ks], d);
                        float o[4];
#pragma unroll
                        for (int v = 0; v < 4; ++v) o[v] = clamp_act(d[v], lo1, hi1);
                        // channels past E have zero weights and bias: they
                        // store zeros, which the depthwise reads with zero taps
                        io<T>::store4(&L.h1r[nq[j]][m * 16 + 4 * g], o);
                    }
                }
            }
            __syncthreads();
            // ---- 3b. depthwise at the active positions + projection slice;
            // meanwhile the next slice's expansion weights go to LDS
            if (ec + 1 < nchunks) stA.store(L.we, C, tid);
            if (ec + 2 < nchunks) stA.load(w1, b1, C, E, ec + 2, tid);
            const int e8 = ec * kChunk + 8 * g;
            const bool ein = e8 < E;
            float bk[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) bk[u] = L.wd.b2[8 * g + u];
            typename M::frag a3[MAXMT];
#pragma unroll
            for (int mt = 0; mt < MAXMT; ++mt) {
                const int c = mt * 16 + r;
                a3[mt] = (ein && c < C) ? M::load(&L.wd.w3[c][8 * g]) : M::zero();
            }
            const char *h1base = reinterpret_cast<const char *>(&L.h1r[0][8 * g]);
#pragma unroll
            for (int j = 0; j < kActTiles; ++j) {
                const int t = wave + NW * j;
                if (t * 16 < n_act) {
                    // every lane computes: a lane past the active list reads
                    // around an own slot and its column of the projection is
                    // never stored (MFMA output columns depend only on their
                    // own B column); channels past E come out as exact zeros
                    float hv[8];
                    {
                        const char *own = h1base + (aq[j] >= 0 ? aq[j] : WP + 1) * col_bytes;
                        // all nine taps in flight before the first FMA
                        typename io<T>::vec8 tv[9];
#pragma unroll
                        for (int k = 0; k < 9; ++k) {
                            const int off = (k / 3 - 1) * row_bytes + (k % 3 - 1) * col_bytes;
                            tv[k] = io<T>::raw8(reinterpret_cast<const T *>(own + off));
                        }
                        float s[8];
#pragma unroll
                        for (int u = 0; u < 8; ++u) s[u] = bk[u];
#pragma unroll
                        for (int k = 0; k < 9; ++k) {
                            // the lane's 8 channels of tap k (4 addresses per wave)
                            const typename io<T>::vec8 wk = io<T>::raw8(&L.wd.w2[k][8 * g]);
#pragma unroll
                            for (int u = 0; u < 8; ++u)
                                s[u] = __builtin_fmaf(static_cast<float>(wk[u]),
                                                      static_cast<float>(tv[k][u]), s[u]);
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
        // ---- 4a. residual sum at the active positions, in place in xs
#pragma unroll
        for (int j = 0; j < kActTiles; ++j) {
            if (aq[j] >= 0) {
#pragma unroll
                for (int mt = 0; mt < MAXMT; ++mt) {
                    const int c0 = mt * 16 + 4 * g;
                    if (c0 < C) {
                        float xv[4], o[4];
                        io<T>::load4(&L.xs[aq[j]][c0], xv);
#pragma unroll
                        for (int v = 0; v < 4; ++v) o[v] = xv[v] + clamp_act(acc[j][mt][v], lo3, hi3);
                        io<T>::store4(&L.xs[aq[j]][c0], o);
                    }
                }
            }
        }
        __syncthreads();
    }
    // ---- 4b. store the patch (inactive positions: x unchanged)
    if (SHUF) {
        // output rows: (first input half, block output) interleaved
        typedef T pair_t __attribute__((ext_vector_type(2)));
        const int nslot = rows_out * cols_out * MAXC;
        for (int i = tid; i < nslot; i += NT) {
            const int pos = i / MAXC, k = i % MAXC;
            if (k < cb) {
                const int rr = 1 + pos / cols_out, c = 1 + pos % cols_out;
                const int64_t g = (img + h0 - 1 + rr) * W + (w0 - 1 + c);
                pair_t v;
                v.x = L.x1s[pos][k];
                v.y = L.xs[rr * WP + c][k];
                *reinterpret_cast<pair_t *>(yout + g * (2 * cb) + 2 * k) = v;
            }
        }
    } else {
        const int vpr = C / per16;
        const int per_row = cols_out * vpr;
        const int nvec = rows_out * per_row;
        for (int i = tid; i < nvec; i += NT) {
            const int rr = 1 + i / per_row, k = i % per_row;
            const int c = 1 + k / vpr, piece = k % vpr;
            uint4 *dst = reinterpret_cast<uint4 *>(yout + ((img + h0 - 1 + rr) * W + (w0 - 1 + c)) * C);
            dst[piece] = *reinterpret_cast<const uint4 *>(&L.xs[rr * WP + c][piece * per16]);
        }
    }
    // ---- 4c. the next block's mask unit on the stored values
    if (!SHUF && mask_next) {
        for (int i = tid; i < rows_out * cols_out; i += NT) {
            const int rr = 1 + i / cols_out, c = 1 + i % cols_out;
            const T *row = &L.xs[rr * WP + c][0];
            float a = 0.0f;
            for (int c0 = 0; c0 < C; c0 += 8) {
                float v[8];
                io<T>::load8(row + c0, v);
#pragma unroll
                for (int u = 0; u < 8; ++u) a = __builtin_fmaf(wm_next[c0 + u], v[u], a);
            }
            const float m = a + bm_next;
            mask_next[(img + h0 - 1 + rr) * W + (w0 - 1 + c)] = mask_decision(m, mask_mode) ? 1 : 0;
        }
    }
}

// counts[2b], counts[2b+1] = sums of the per-patch counts of block b
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
        if (static_cast<int>(threadIdx.x) < off) {
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
