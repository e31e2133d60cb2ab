// cells.h -- work-balanced one-launch gated block for narrow blocks (gfx950).
//
// k_block_cells runs a whole spatially gated inverted-residual block (Sec.
// 3.2) for blocks of at most 32 channels and 192 hidden channels in 16-bit
// storage.  The image is cut into cells of 2 x 8 positions; one wave owns a
// cell from start to end, with no barrier between waves:
//   1. x and the hard-mask bytes of the cell's 4 x 10 region (the cell plus a
//      one-position ring) are read in one round trip: x into the wave's LDS
//      copy of the region, the mask into one 64-bit ballot word.  The cell's
//      active set and the part of its 3x3 dilation inside the region (every
//      in-image region position next to an active one) follow by shifts of
//      that word, and their raster-ordered lists by popcount ranks;
//   2. for each 32-channel slice of the hidden layer: expansion of the
//      needed positions on the matrix cores (the bias is the accumulator's
//      start), activation, stored at the position's slot of the wave's
//      region array (slots outside the image hold zeros: the depthwise
//      padding); the depthwise 3x3 at the active positions reads its 9 taps
//      at fixed slot offsets; its output is the B operand of the projection,
//      accumulated over the slices on the matrix cores;
//   3. epilogue: y = x + F at the active positions, x elsewhere, stored for
//      every position of the cell; then the next block's mask unit on the
//      stored values (the fp32 multiply-add chain of k_mask), and the
//      cell's active count for the next launch's schedule.
// Every weight of the block sits in LDS for the whole launch.  The grid is
// persistent (one workgroup of 16 waves per CU).  The active cells, ranked
// in raster order from the per-cell counts that the previous launch wrote,
// are dealt to the workgroups in equal shares by count; they go to the 16
// waves in turn (so they spread evenly over the SIMDs), each wave finding
// the cell of its rank by ballots over the counts, and the waves then
// stream, through a counter in LDS, the empty cells of the workgroup's equal
// share of the grid (copy and next mask unit, one position per lane), so
// the copies overlap the active work of the other waves.  A dense region of
// the mask is spread over many CUs, and the span follows the active work.
// The arithmetic of every output element is the one of the kernel chain
// (k_expand, k_dw_project): the same operand fragments, summation order and
// roundings.  Input and output must be different buffers (a cell's ring is
// another cell's output).
#pragma once

#include "fused.h"

namespace dynconv {

// A cell is 2 image rows x 8 columns: 16 own positions, one 16-position tile
// of the depthwise / projection, and a 4 x 10 region (the cell plus its ring)
// of at most 40 positions, so one 64-bit ballot holds the region's mask.
constexpr int kCellRows = 2, kCellCols = 8;
constexpr int kCellOwn = kCellRows * kCellCols;       // 16 own positions
constexpr int kRegCols = kCellCols + 2;               // 10
constexpr int kRegRows = kCellRows + 2;               // 4
constexpr int kRegSlots = kRegRows * kRegCols;        // 40 region slots
constexpr int kNeedTiles = (kRegSlots + 15) / 16;     // 3
constexpr int kCellWaves = 16;                        // 4 waves per SIMD: 128 registers
constexpr int kCellThreads = kCellWaves * kWave;
constexpr int kCellMaxC = 32;
constexpr int kCellMaxE = 192;
constexpr int kCellFirstOwn = kRegCols + 1;           // slot of own position (0, 0)

// Region slots (row rr, column cc) -> bit rr*10 + cc.
constexpr uint64_t kRowBits = 0xffull << 1;           // columns 1..8 of one region row
constexpr uint64_t kOwnBits = (kRowBits << 10) | (kRowBits << 20);
constexpr uint64_t kCol0Bits = 1ull | (1ull << 10) | (1ull << 20) | (1ull << 30);
constexpr uint64_t kCol9Bits = kCol0Bits << 9;

__host__ __device__ inline int cells_per_image(int H, int W) {
    return ((H + kCellRows - 1) / kCellRows) * ((W + kCellCols - 1) / kCellCols);
}

template <typename T>
struct CellWeights {
    alignas(16) T w1[kCellMaxE][kCellMaxC + 8];   // expansion rows e, channels fastest (zero past C, E)
    alignas(16) T w3[kCellMaxC][kCellMaxE + 8];   // projection rows c, hidden fastest (zero past C, E)
    alignas(16) T w2[9][kCellMaxE + 8];           // depthwise taps, transposed (zero past E); the
                                                  // padding puts the nine rows on distinct LDS banks
    alignas(16) float b1[kCellMaxE];
    alignas(16) float b2[kCellMaxE];
    alignas(16) float b3[kCellMaxC];
    alignas(16) float wm[kCellMaxC];              // the next block's mask unit
};

// A slice of the expansion in region layout: slot (rr, cc) at byte
// rr * kRegPitch + cc * kSlotBytes.  The 96 padding bytes per region row put
// the two image rows of a 16-position tile on distinct LDS banks (a 16-byte
// read of 16 lanes touches every bank once); a spare slot at the end takes
// the padding lanes of the last tile.
constexpr int kSlotBytes = kChunkPad * 2;                 // 80: 32 channels + 8 padding, 16-bit
constexpr int kRegPitch = kRegCols * kSlotBytes + 96;     // 896
constexpr int kSpareSlot = kRegRows * kRegPitch;          // byte offset of the spare slot
__device__ __forceinline__ int slot_off(int q) { return (q / kRegCols) * kRegPitch + (q % kRegCols) * kSlotBytes; }

template <typename T>
struct CellWaveLds {
    alignas(16) char h1[kSpareSlot + kSlotBytes];  // the region array of one slice
    alignas(16) T xr[kRegSlots][kChunkPad];        // x at the region slots; the own slots become y
    int8_t need[48];
    int8_t act[kCellOwn];
};

// Lane S of each 16-lane row of the wave, to every lane of that row (DPP
// row_newbcast, one move per register).
template <int S>
__device__ __forceinline__ uint4 row_bcast16(uint4 v) {
    static_assert(S >= 0 && S < 16, "source lane within the row");
    uint4 o;
    o.x = __builtin_amdgcn_mov_dpp(v.x, 0x150 + S, 0xf, 0xf, false);
    o.y = __builtin_amdgcn_mov_dpp(v.y, 0x150 + S, 0xf, 0xf, false);
    o.z = __builtin_amdgcn_mov_dpp(v.z, 0x150 + S, 0xf, 0xf, false);
    o.w = __builtin_amdgcn_mov_dpp(v.w, 0x150 + S, 0xf, 0xf, false);
    return o;
}

// A 16-byte store that the next launch reads, not this one: nontemporal, so
// that the lines leave the L2 as they are written rather than at the end of
// the launch.
__device__ __forceinline__ void store_stream(uint4 *dst, uint4 v) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4 *>(dst));
}

// Stream work unit: 4 cells (64 positions, one per lane).
constexpr int kStreamCells = kWave / kCellOwn;

template <typename T>
struct CellLds {
    CellWeights<T> w;
    CellWaveLds<T> wv[kCellWaves];
    // per thread: its wave's inclusive active-cell count up to and including
    // the thread's chunks of the count buffer, and the active bits of its
    // (first) chunk
    uint2 tab[kCellThreads];
    int part[kCellWaves];
    int next, next_stream;
};

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
}

// mask unit (Eq. 2, Eq. 8 at zero noise) on one stored row: the fp32
// multiply-add chain of k_mask, channels ascending from +0, then the bias
constexpr int kCellPieces = kCellMaxC * 2 / 16;   // 16-byte pieces of a 16-bit row

template <typename T>
__device__ __forceinline__ bool cell_mask_row(const uint4 (&row)[kCellPieces], const float *wm, int C, float bm,
                                              int mode) {
    constexpr int per16 = 16 / static_cast<int>(sizeof(T));
    float a = 0.0f;
#pragma unroll
    for (int p = 0; p < kCellPieces; ++p) {
        if (p < C / per16) {
            float v[8];
            io<T>::load8(reinterpret_cast<const T *>(&row[p]), v);
#pragma unroll
            for (int u = 0; u < 8; ++u) a = __builtin_fmaf(wm[p * per16 + u], v[u], a);
        }
    }
    return mask_decision(a + bm, mode);
}

// Popcount of this lane's 16-lane group in a ballot (the group is one cell).
__device__ __forceinline__ int group16_count(uint64_t b, int lane) {
    return __popc(static_cast<uint32_t>((b >> (lane & 48)) & 0xffffull));
}

// Bit b (b < 4) set where byte b of w is nonzero: the top bit of each byte of
// ((w & 0x7f7f7f7f) + 0x7f7f7f7f) | w, the four gathered by one multiply
// (the partial products land on distinct bits, none of them in 21..24).
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {
    const uint32_t h = (((w & 0x7f7f7f7fu) + 0x7f7f7f7fu) | w) & 0x80808080u;
    return (((h >> 7) * 0x00204081u) >> 21) & 0xfu;
}

// floor(k * total / G) for 0 <= k <= G and 0 <= total <= the cell count: the
// host launches the kernel only when the cell count times G fits in 32 bits.
__device__ __forceinline__ int share_bound(int k, int total, int G) {
    return static_cast<int>(static_cast<uint32_t>(k) * static_cast<uint32_t>(total) / static_cast<uint32_t>(G));
}

// The first block's mask unit over cells: mask bytes of every position and
// each cell's active count (four cells per wave, lane = own position).
constexpr int kCellsPerMaskWave = kWave / kCellOwn;

template <typename T>
__global__ void __launch_bounds__(kBlock)
k_mask_cells(const T *__restrict__ x, int N, int H, int W, int C, const float *__restrict__ wm, float bm,
             uint8_t *__restrict__ mask, uint8_t *__restrict__ cell_cnt, int mode) {
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int ncw = (W + kCellCols - 1) / kCellCols;
    const int cpi = cells_per_image(H, W);
    const int64_t ncells = static_cast<int64_t>(N) * cpi;
    const int64_t c = (static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + wave) * kCellsPerMaskWave + lane / kCellOwn;
    const int o = lane % kCellOwn;
    bool bit = false;
    if (c < ncells) {
        const int n = static_cast<int>(c / cpi), rem = static_cast<int>(c % cpi);
        const int h = (rem / ncw) * kCellRows + o / kCellCols;
        const int w = (rem % ncw) * kCellCols + o % kCellCols;
        if (h < H && w < W) {
            const int64_t pos = (static_cast<int64_t>(n) * H + h) * W + w;
            uint4 row[kCellPieces];
            const uint4 *src = reinterpret_cast<const uint4 *>(x + pos * C);
#pragma unroll
            for (int p = 0; p < kCellPieces; ++p)
                row[p] = (p < C * static_cast<int>(sizeof(T)) / 16) ? src[p] : make_uint4(0, 0, 0, 0);
            bit = cell_mask_row<T>(row, wm, C, bm, mode);
            mask[pos] = bit ? 1 : 0;
        }
    }
    const uint64_t b = __ballot(bit);
    if (c < ncells && o == 0) cell_cnt[c] = static_cast<uint8_t>(group16_count(b, lane));
}

template <typename T, bool DENSE>
__global__ void __launch_bounds__(kCellThreads)
k_block_cells(const T *__restrict__ xin, T *__restrict__ yout, int N, int H, int W, int C, int E, int G,
              const uint8_t *__restrict__ mask_in, const uint8_t *__restrict__ cnt_in,
              const T *__restrict__ w1, const float *__restrict__ b1, int act1,
              const T *__restrict__ w2, const float *__restrict__ b2, int act2,
              const T *__restrict__ w3, const float *__restrict__ b3, int act3,
              const float *__restrict__ wm_next, float bm_next, uint8_t *__restrict__ mask_next,
              uint8_t *__restrict__ cnt_next, int32_t *__restrict__ band_counts, int mask_mode) {
    typedef mma<T> M;
    constexpr int per16 = 16 / static_cast<int>(sizeof(T));
    __shared__ CellLds<T> L;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const int r = lane % 16, g = lane / 16;
    // XCD-aware: workgroup b runs on XCD b % 8 and takes share k, so each XCD
    // holds a contiguous run of shares (cells next to each other share rings)
    const int per_xcd = (G + 7) / 8;
    const int k = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (k >= G) return;  // uniform per workgroup
    const int ncw = (W + kCellCols - 1) / kCellCols;
    const int cpi = cells_per_image(H, W);
    const int ncells = N * cpi;
    const int E32 = (E + kChunk - 1) / kChunk * kChunk;

    // this thread's chunks of the count buffer (16 cells per 16-byte word; the
    // count buffers are padded to whole 256 bytes); the first chunk is
    // requested before the weights, so both latencies overlap
    const int nchunks = (ncells + 15) / 16;
    const int per = (nchunks + kCellThreads - 1) / kCellThreads;
    const int q0 = tid * per, q1 = min(q0 + per, nchunks);
    auto active_bits = [&](uint4 v, int i) {  // bit u: cell i + u (< ncells) is active
        const uint32_t bits = nonzero_bytes(v.x) | (nonzero_bytes(v.y) << 4) | (nonzero_bytes(v.z) << 8) |
                              (nonzero_bytes(v.w) << 12);
        const int left = ncells - i;
        return (left >= 16) ? bits : bits & ((1u << left) - 1u);
    };
    uint4 first_raw = make_uint4(0, 0, 0, 0);
    if (!DENSE && q0 < q1) first_raw = reinterpret_cast<const uint4 *>(cnt_in)[q0];

    // ---- all weights of the block into LDS (zero past C and E): every
    // thread's global loads are issued before its LDS stores
    {
        constexpr int kW1 = kCellMaxE * (kCellMaxC / 8), kW3 = kCellMaxC * (kCellMaxE / 8);
        constexpr int kS1 = (kW1 + kCellThreads - 1) / kCellThreads, kS3 = (kW3 + kCellThreads - 1) / kCellThreads;
        constexpr int kS2 = (kCellMaxE * 9 + kCellThreads - 1) / kCellThreads;
        uint4 v1[kS1], v3[kS3];
        T v2[kS2];
#pragma unroll
        for (int sl = 0; sl < kS1; ++sl) {
            const int i = tid + sl * kCellThreads;
            const int e = i / (kCellMaxC / 8), c8 = (i % (kCellMaxC / 8)) * 8;
            v1[sl] = (e < E && c8 < C) ? *reinterpret_cast<const uint4 *>(w1 + static_cast<int64_t>(e) * C + c8)
                                       : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int sl = 0; sl < kS3; ++sl) {
            const int i = tid + sl * kCellThreads;
            const int c = i / (kCellMaxE / 8), e8 = (i % (kCellMaxE / 8)) * 8;
            v3[sl] = (c < C && e8 < E) ? *reinterpret_cast<const uint4 *>(w3 + static_cast<int64_t>(c) * E + e8)
                                       : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int sl = 0; sl < kS2; ++sl) {
            const int j = tid + sl * kCellThreads;
            v2[sl] = (j < E * 9) ? w2[j] : static_cast<T>(0.0f);
        }
        float vb1 = 0.0f, vb2 = 0.0f, vb3 = 0.0f, vwm = 0.0f;
        if (tid < kCellMaxE) {
            vb1 = (tid < E) ? b1[tid] : 0.0f;
            vb2 = (tid < E) ? b2[tid] : 0.0f;
        }
        if (tid < kCellMaxC) {
            vb3 = (tid < C) ? b3[tid] : 0.0f;
            vwm = (wm_next && tid < C) ? wm_next[tid] : 0.0f;
        }
#pragma unroll
        for (int sl = 0; sl < kS1; ++sl) {
            const int i = tid + sl * kCellThreads;
            if (i < kW1) *reinterpret_cast<uint4 *>(&L.w.w1[i / (kCellMaxC / 8)][(i % (kCellMaxC / 8)) * 8]) = v1[sl];
        }
#pragma unroll
        for (int sl = 0; sl < kS3; ++sl) {
            const int i = tid + sl * kCellThreads;
            if (i < kW3) *reinterpret_cast<uint4 *>(&L.w.w3[i / (kCellMaxE / 8)][(i % (kCellMaxE / 8)) * 8]) = v3[sl];
        }
#pragma unroll
        for (int sl = 0; sl < kS2; ++sl) {
            const int j = tid + sl * kCellThreads;
            if (j < kCellMaxE * 9) L.w.w2[j % 9][j / 9] = v2[sl];
        }
        if (tid < kCellMaxE) {
            L.w.b1[tid] = vb1;
            L.w.b2[tid] = vb2;
        }
        if (tid < kCellMaxC) {
            L.w.b3[tid] = vb3;
            L.w.wm[tid] = vwm;
        }
    }

    // ---- this workgroup's work.  Dense: cells [u_lo, u_hi), an equal share.
    // Gated: the active cells are dealt in equal shares by count (share k is
    // the active cells with rank [a_lo, a_hi) in raster order, ranked from
    // the per-cell active counts that the previous launch wrote), and the
    // empty cells of [u_lo, u_hi) are streamed (a copy and the next mask
    // unit: memory-bound, no ring needed) once a wave runs out of active
    // cells.  So a dense region of the mask is spread over many CUs, and the
    // span follows the active work.  One barrier: the weights, the ranks and
    // the counters.
    const int u_lo = share_bound(k, ncells, G);
    const int u_hi = share_bound(k + 1, ncells, G);
    if (!DENSE) {
        const uint32_t first = (q0 < q1) ? active_bits(first_raw, q0 * 16) : 0u;
        int cnt = __popc(first);
        for (int q = q0 + 1; q < q1; ++q)
            cnt += __popc(active_bits(reinterpret_cast<const uint4 *>(cnt_in)[q], q * 16));
        const int incl = wave_scan_incl(cnt);
        L.tab[tid] = make_uint2(static_cast<uint32_t>(incl), first);
        if (lane == kWave - 1) L.part[wave] = incl;
    }
    if (tid == 0) {
        L.next = 0;
        L.next_stream = 0;
    }
    __syncthreads();
    // gated: the waves' inclusive counts in lanes 0..15, the share's ranks
    int pw = 0, a_lo = 0, a_hi = u_hi - u_lo;
    if (!DENSE) {
        pw = wave_scan_incl(lane < kCellWaves ? L.part[lane] : 0);
        const int total = __builtin_amdgcn_readlane(pw, kCellWaves - 1);
        a_lo = share_bound(k, total, G);
        a_hi = share_bound(k + 1, total, G);
    }
    // the bounds are the same in every lane: keep them in scalar registers,
    // so that the loops below are uniform control flow (with a bound in a
    // vector register the compiler may split a loop per lane, and lanes
    // other than lane 0 would then reread a counter's start)
    a_lo = __builtin_amdgcn_readfirstlane(a_lo);
    a_hi = __builtin_amdgcn_readfirstlane(a_hi);
    const int n_stream = DENSE ? 0 : (u_hi - u_lo + kStreamCells - 1) / kStreamCells;

    const float lo1 = act_lo(act1), hi1 = act_hi(act1);
    const float lo2 = act_lo(act2), hi2 = act_hi(act2);
    const float lo3 = act_lo(act3), hi3 = act_hi(act3);
    const int nsl = E32 / kChunk;
    const int npieces = C / per16;
    const int rr = lane / kRegCols, cc = lane % kRegCols;    // this lane's region slot
    const int oi = lane / kCellCols, oj = lane % kCellCols;  // this lane's own position (lane < 16)
    const int oslot = (oi + 1) * kRegCols + oj + 1;          // ... and its region slot
    const uint64_t lt = lanemask_lt(lane);
    CellWaveLds<T> &V = L.wv[wave];

    // One active cell (gated) or any cell (dense), by one wave.
    auto run_cell = [&](int cell) {
        // Gated: a wave's issue priority falls as its cell progresses (3 for
        // the region and the first two slices, 2 for the next two, 1 for the
        // last two, 0 after the cell).  The SIMD's issue arbiter favours the
        // oldest wave among those of the highest priority, so without this
        // the third cell on a SIMD ran behind the other two and finished
        // alone, latency-bound; with it the cells of a SIMD progress together
        // and the streaming waves (priority 0) fill the gaps.
        if (!DENSE) __builtin_amdgcn_s_setprio(3);
        const int n = cell / cpi, rem = cell % cpi;
        const int h0 = (rem / ncw) * kCellRows, w0 = (rem % ncw) * kCellCols;
        const int64_t img = static_cast<int64_t>(n) * H;

        // ---- 1. x and the mask at the region slots in one round trip; the
        // region's mask word, active set, needed set, lists
        const int hh = h0 - 1 + rr, ww = w0 - 1 + cc;
        const bool inimg = lane < kRegSlots && hh >= 0 && hh < H && ww >= 0 && ww < W;
        bool mb = false;
        if (inimg) {
            const int64_t gp = (img + hh) * W + ww;
            const uint4 *src = reinterpret_cast<const uint4 *>(xin + gp * C);
            uint4 xv[kCellPieces];
#pragma unroll
            for (int p = 0; p < kCellPieces; ++p) xv[p] = (p < npieces) ? src[p] : make_uint4(0, 0, 0, 0);
            mb = DENSE ? true : (mask_in[gp] != 0);
#pragma unroll
            for (int p = 0; p < kCellPieces; ++p)
                if (p < npieces) reinterpret_cast<uint4 *>(&V.xr[lane][0])[p] = xv[p];
        }
        const uint64_t IMG = __ballot(inimg);
        const uint64_t Gw = __ballot(mb);
        const uint64_t A = Gw & kOwnBits;
        uint64_t Dw = A | (A << 1) | (A >> 1);     // own columns 1..8: no row wrap
        Dw |= (Dw << kRegCols) | (Dw >> kRegCols);
        const uint64_t NEED = Dw & IMG;
        if (!DENSE && band_counts) {
            // the cell's active and dilated counts (its own positions whose 3x3
            // neighbourhood holds an active position of any cell)
            uint64_t Gd = Gw | ((Gw << 1) & ~kCol0Bits) | ((Gw >> 1) & ~kCol9Bits);
            Gd |= (Gd << kRegCols) | (Gd >> kRegCols);
            Gd &= kOwnBits & IMG;
            *reinterpret_cast<int2 *>(band_counts + 2 * static_cast<int64_t>(cell)) =
                make_int2(__popcll(A), __popcll(Gd));  // the same value from every lane
        }
        const int oh = h0 + oi, ow = w0 + oj;
        const bool ov = lane < kCellOwn && oh < H && ow < W;

        if (A != 0) {
            const int nneed = __popcll(NEED);
            const int ntn = (nneed + 15) >> 4;
            if ((NEED >> lane) & 1ull) V.need[__popcll(NEED & lt)] = static_cast<int8_t>(lane);
            if ((A >> lane) & 1ull) V.act[__popcll(A & lt)] = static_cast<int8_t>(lane);
            if (lane < kRegSlots && !inimg) {  // the depthwise's zero padding
                uint4 *z = reinterpret_cast<uint4 *>(V.h1 + slot_off(lane));
#pragma unroll
                for (int p = 0; p < kChunk * 2 / 16; ++p) z[p] = make_uint4(0, 0, 0, 0);
            }
            wave_sync();
            // needed slots (the expansion's output rows, as byte offsets;
            // padding lanes: the spare slot) and their B fragments, kept for
            // every slice
            int nq[kNeedTiles];
            typename M::frag bx[kNeedTiles];
#pragma unroll
            for (int t = 0; t < kNeedTiles; ++t) {
                const int i = 16 * t + r;
                const int q = (i < nneed) ? static_cast<int>(V.need[i]) : -1;
                nq[t] = (q >= 0) ? slot_off(q) : kSpareSlot;
                const int qx = (q >= 0) ? q : kCellFirstOwn;  // an in-image slot
                bx[t] = (t < ntn && 8 * g < C) ? M::load(&V.xr[qx][8 * g]) : M::zero();
            }
            // the tile's active position of this lane (padding lanes: -1)
            const int aq = (r < __popcll(A)) ? static_cast<int>(V.act[r]) : -1;
            floatx4 acc[2];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[mt][v] = L.w.b3[mt * 16 + 4 * g + v];
            // padding lanes compute around an own slot; their projection
            // columns are never stored
            const char *own = V.h1 + slot_off(aq >= 0 ? aq : kCellFirstOwn) + 16 * g;

            for (int ec = 0; ec < nsl; ++ec) {
                const int eb = ec * kChunk;
                if (!DENSE) {
                    if (ec == 2) __builtin_amdgcn_s_setprio(2);
                    else if (ec == 4) __builtin_amdgcn_s_setprio(1);
                }
                // ---- 2a. expansion of the needed slots into the region array:
                // the tiles' products issued back to back, then activated
                // the slice's per-channel constants.  Dense launches (four busy
                // waves per SIMD, the LDS the tighter resource): one 16-byte
                // read per lane (lane r of a 16-lane row: tap r's depthwise
                // weights for r < 9, the depthwise bias for r = 9, 10, the
                // expansion bias of the two output tiles for r = 11, 12),
                // broadcast within the row by DPP moves.  Gated launches (about
                // three busy waves per SIMD, the vector ALU the tighter
                // resource): row-wide broadcast reads from LDS instead, with
                // no vector instruction.  The values are the same.
                const uint4 pk = !DENSE ? make_uint4(0, 0, 0, 0) : *reinterpret_cast<const uint4 *>(
                    r < 9 ? reinterpret_cast<const char *>(&L.w.w2[r][eb + 8 * g])
                    : r < 11 ? reinterpret_cast<const char *>(&L.w.b2[eb + 8 * g + 4 * (r - 9)])
                             : reinterpret_cast<const char *>(&L.w.b1[eb + 16 * (r == 12) + 4 * g]));
                typename M::frag a1[2];
                floatx4 bi[2];
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    a1[m] = M::load(&L.w.w1[eb + m * 16 + r][8 * g]);
                    if (!DENSE) {
                        bi[m] = *reinterpret_cast<const floatx4 *>(&L.w.b1[eb + m * 16 + 4 * g]);
                    } else {
                        const uint4 b = (m == 0) ? row_bcast16<11>(pk) : row_bcast16<12>(pk);
                        bi[m][0] = __uint_as_float(b.x);
                        bi[m][1] = __uint_as_float(b.y);
                        bi[m][2] = __uint_as_float(b.z);
                        bi[m][3] = __uint_as_float(b.w);
                    }
                }
                auto expand = [&](auto ntiles) {
                    constexpr int NTL = decltype(ntiles)::value;
                    floatx4 d[NTL][2];
#pragma unroll
                    for (int t = 0; t < NTL; ++t)
#pragma unroll
                        for (int m = 0; m < 2; ++m) d[t][m] = M::run(a1[m], bx[t], bi[m]);
#pragma unroll
                    for (int t = 0; t < NTL; ++t)
#pragma unroll
                        for (int m = 0; m < 2; ++m) {
                            float o[4];
#pragma unroll
                            for (int v = 0; v < 4; ++v) o[v] = clamp_act(d[t][m][v], lo1, hi1);
                            // a tile past the needed ones stores into the spare slot
                            io<T>::store4(reinterpret_cast<T *>(V.h1 + nq[t]) + m * 16 + 4 * g, o);
                        }
                };
                if (ntn == 3) expand(std::integral_constant<int, 3>());
                else if (ntn == 2) expand(std::integral_constant<int, 2>());
                else expand(std::integral_constant<int, 1>());
                wave_sync();
                // ---- 2b. depthwise at the tile's positions + projection slice
                typename M::frag a3[2];
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) a3[mt] = M::load(&L.w.w3[mt * 16 + r][eb + 8 * g]);
                // all nine taps and their weights requested before the first
                // multiply-add (the LDS latency is paid once per slice)
                typename io<T>::vec8 tv[9];
#pragma unroll
                for (int t = 0; t < 9; ++t)
                    tv[t] = io<T>::raw8(reinterpret_cast<const T *>(
                        own + (t / 3 - 1) * kRegPitch + (t % 3 - 1) * kSlotBytes));
                float s[8];
                if (!DENSE) {
                    const floatx4 lo = *reinterpret_cast<const floatx4 *>(&L.w.b2[eb + 8 * g]);
                    const floatx4 hi = *reinterpret_cast<const floatx4 *>(&L.w.b2[eb + 8 * g + 4]);
                    s[0] = lo[0]; s[1] = lo[1]; s[2] = lo[2]; s[3] = lo[3];
                    s[4] = hi[0]; s[5] = hi[1]; s[6] = hi[2]; s[7] = hi[3];
                } else {
                    const uint4 lo = row_bcast16<9>(pk), hi = row_bcast16<10>(pk);
                    s[0] = __uint_as_float(lo.x); s[1] = __uint_as_float(lo.y);
                    s[2] = __uint_as_float(lo.z); s[3] = __uint_as_float(lo.w);
                    s[4] = __uint_as_float(hi.x); s[5] = __uint_as_float(hi.y);
                    s[6] = __uint_as_float(hi.z); s[7] = __uint_as_float(hi.w);
                }
                auto tap = [&](auto t) {
                    constexpr int TT = decltype(t)::value;
                    const uint4 wb = !DENSE ? *reinterpret_cast<const uint4 *>(&L.w.w2[TT][eb + 8 * g])
                                            : row_bcast16<TT>(pk);
                    const typename io<T>::vec8 wk = *reinterpret_cast<const typename io<T>::vec8 *>(&wb);
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        s[u] = __builtin_fmaf(static_cast<float>(wk[u]), static_cast<float>(tv[TT][u]), s[u]);
                };
                tap(std::integral_constant<int, 0>());
                tap(std::integral_constant<int, 1>());
                tap(std::integral_constant<int, 2>());
                tap(std::integral_constant<int, 3>());
                tap(std::integral_constant<int, 4>());
                tap(std::integral_constant<int, 5>());
                tap(std::integral_constant<int, 6>());
                tap(std::integral_constant<int, 7>());
                tap(std::integral_constant<int, 8>());
                float hv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) hv[u] = clamp_act(s[u], lo2, hi2);
                const typename M::frag bf = M::pack(hv);
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) acc[mt] = M::run(a3[mt], bf, acc[mt]);
                wave_sync();
            }

            // ---- 3a. residual sum at the active positions, in place on the
            // staged own rows
            if (aq >= 0) {
#pragma unroll
                for (int mt = 0; mt < 2; ++mt) {
                    const int c0 = mt * 16 + 4 * g;
                    if (c0 < C) {
                        float xv[4], out[4];
                        io<T>::load4(&V.xr[aq][c0], xv);
#pragma unroll
                        for (int v = 0; v < 4; ++v) out[v] = xv[v] + clamp_act(acc[mt][v], lo3, hi3);
                        io<T>::store4(&V.xr[aq][c0], out);
                    }
                }
            }
        }
        wave_sync();

        // ---- 3b. store the cell, the next block's mask unit on the stored values
        uint4 yr[kCellPieces];
#pragma unroll
        for (int p = 0; p < kCellPieces; ++p)
            yr[p] = (ov && p < npieces) ? reinterpret_cast<const uint4 *>(&V.xr[oslot][0])[p] : make_uint4(0, 0, 0, 0);
        wave_sync();  // the staged rows are read before the next cell overwrites them
        if (ov) {
            uint4 *dst = reinterpret_cast<uint4 *>(yout + ((img + oh) * W + ow) * C);
#pragma unroll
            for (int p = 0; p < kCellPieces; ++p)
                if (p < npieces) store_stream(&dst[p], yr[p]);
        }
        if (!DENSE && mask_next) {
            bool bit = false;
            if (ov) {
                bit = cell_mask_row<T>(yr, L.w.wm, C, bm_next, mask_mode);
                mask_next[(img + oh) * W + ow] = bit ? 1 : 0;
            }
            const uint64_t b = __ballot(bit);
            cnt_next[cell] = static_cast<uint8_t>(__popcll(b));  // the same value from every lane
        }
        if (!DENSE) __builtin_amdgcn_s_setprio(0);
    };

    // Four empty cells of [u_lo, u_hi) (chunk j), one position per lane:
    // y = x, the next block's mask unit, the cells' counts.
    auto run_stream = [&](int j) {
        const int i = j * kWave + lane;
        const int cell = u_lo + i / kCellOwn;
        const bool empty = cell < u_hi && cnt_in[cell] == 0;
        const int o = i % kCellOwn;
        const int rem = cell % cpi;
        const int h = (rem / ncw) * kCellRows + o / kCellCols;
        const int w = (rem % ncw) * kCellCols + o % kCellCols;
        const bool take = empty && h < H && w < W;
        const int64_t img = static_cast<int64_t>(cell / cpi) * H;
        const int64_t pos = (img + h) * W + w;
        uint4 row[kCellPieces];
#pragma unroll
        for (int p = 0; p < kCellPieces; ++p)
            row[p] = (take && p < npieces) ? reinterpret_cast<const uint4 *>(xin + pos * C)[p] : make_uint4(0, 0, 0, 0);
        if (take) {
            uint4 *dst = reinterpret_cast<uint4 *>(yout + pos * C);
#pragma unroll
            for (int p = 0; p < kCellPieces; ++p)
                if (p < npieces) store_stream(&dst[p], row[p]);
        }
        bool bit = false;
        if (take && mask_next) {
            bit = cell_mask_row<T>(row, L.w.wm, C, bm_next, mask_mode);
            mask_next[pos] = bit ? 1 : 0;
        }
        const int cnt = group16_count(__ballot(bit), lane);
        if (empty && mask_next) cnt_next[cell] = static_cast<uint8_t>(cnt);
        if (band_counts) {
            // no active position; dilated: own positions next to an active
            // position of a neighbouring cell
            bool dil = false;
            if (take) {
                for (int dh = -1; dh <= 1; ++dh)
                    for (int dw = -1; dw <= 1; ++dw) {
                        const int hh = h + dh, ww = w + dw;
                        if (hh >= 0 && hh < H && ww >= 0 && ww < W && mask_in[(img + hh) * W + ww] != 0) dil = true;
                    }
            }
            const int nd = group16_count(__ballot(dil), lane);
            if (empty) *reinterpret_cast<int2 *>(band_counts + 2 * static_cast<int64_t>(cell)) = make_int2(0, nd);
        }
    };

    // The active cell of rank R (gated): the wave whose chunks hold it (the
    // waves' inclusive counts), the thread within that wave (its inclusive
    // counts in LDS), the chunk of that thread, and the bit within the chunk.
    // Every step is a ballot over the wave, so R, the result and every index
    // on the way are uniform.  With more than one chunk per thread (large
    // batches) the thread's chunks are read again, one per lane, 64 at a
    // time, and a wave scan of their counts picks the chunk.
    auto find = [&](int R) {
        const int v = __popcll(__ballot(lane < kCellWaves && pw <= R));  // waves wholly before R
        const int rv = R - (v > 0 ? __builtin_amdgcn_readlane(pw, v - 1) : 0);
        const uint2 e = L.tab[v * kWave + lane];
        const int t = __popcll(__ballot(static_cast<int>(e.x) <= rv));  // threads wholly before R
        int local = rv - (t > 0 ? static_cast<int>(__builtin_amdgcn_readlane(e.x, t - 1)) : 0);
        int q = (v * kWave + t) * per;
        uint32_t bits = __builtin_amdgcn_readlane(e.y, t);
        if (per > 1) {
            const int q_end = min(q + per, nchunks);
            for (int base = q; base < q_end; base += kWave) {
                const int qq = base + lane;
                const uint32_t b = (qq < q_end) ? active_bits(reinterpret_cast<const uint4 *>(cnt_in)[qq], qq * 16) : 0u;
                const int incl = wave_scan_incl(__popc(b));
                const int j = __popcll(__ballot(incl <= local));  // chunks wholly before
                q = base + j;
                if (j < kWave) {
                    local -= (j > 0 ? __builtin_amdgcn_readlane(incl, j - 1) : 0);
                    bits = __builtin_amdgcn_readlane(b, j);
                    break;
                }
                local -= __builtin_amdgcn_readlane(incl, kWave - 1);
            }
        }
        const bool hit = lane < 16 && ((bits >> lane) & 1u) && __popc(bits & ((1u << lane) - 1u)) == local;
        const uint64_t hb = __ballot(hit);
        // (the counts are read-only in this launch, so a hit always exists; the
        // guards only keep an index in range whatever the data)
        return min(q, nchunks - 1) * 16 + (hb ? __builtin_amdgcn_readfirstlane(__ffsll(static_cast<long long>(hb)) - 1) : 0);
    };

    // Gated: the share's active cells go to the waves in turn (rank a_lo + i
    // to wave i mod kCellWaves).  Wave w runs on SIMD w mod 4, so the cells
    // spread evenly over the SIMDs: with a shared counter, whichever waves
    // come first take them, and one SIMD could hold 4 of a workgroup's 11
    // cells while another holds 2.  Dense: every cell costs the same and a
    // shared counter (one LDS atomic per wave, merged by the compiler) keeps
    // the waves busy.  Bounds, items and the wave index are scalars, so both
    // loops are uniform control flow.
    if (!DENSE) {
        const int wave_s = __builtin_amdgcn_readfirstlane(wave);
        for (int item = a_lo + wave_s; item < a_hi; item += kCellWaves) run_cell(find(item));
        for (;;) {
            const int j = __builtin_amdgcn_readlane(atomicAdd(&L.next_stream, 1), 0) >> 6;
            if (j >= n_stream) break;
            run_stream(j);
        }
    } else {
        for (;;) {
            const int item = __builtin_amdgcn_readlane(atomicAdd(&L.next, 1), 0) >> 6;
            if (item >= a_hi) break;
            run_cell(u_lo + item);
        }
    }
}

}  // namespace dynconv
