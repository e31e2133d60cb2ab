// dynconv.hip -- host side of the C ABI declared in include/dynconv.h:
// argument validation, workspace carving and kernel launches.  Every entry
// point validates everything before it enqueues anything, allocates nothing
// and never synchronises with the host.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <algorithm>
#include <atomic>
#include <string.h>

#include "dynconv.h"
#include "cells.h"
#include "fused.h"
#include "kernels.h"
#include "shuffle.h"
#include "dense.h"

using namespace dynconv;

namespace {

constexpr int kMaxC = 256;
constexpr int kMaxE = 1536;
constexpr int kMaxDilate = 3;
constexpr int kMaxBlocks = 1024;
constexpr int64_t kMaxPositions = (int64_t{1} << 31) / 9 - 1;
constexpr int kMaxGrid = 2048;  // workgroups of the row-tile kernels (grid-stride beyond)
constexpr int kMaxDwGrid = 8192;  // workgroups of the depthwise-projection kernel
constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

size_t dtype_size(dynconv_dtype dt) { return dt == DYNCONV_F32 ? 4 : 2; }

bool dtype_ok(int dt) { return dt == DYNCONV_F32 || dt == DYNCONV_F16 || dt == DYNCONV_BF16; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t positions(dynconv_shape s) {
    return static_cast<int64_t>(s.n) * s.h * s.w;
}

dynconv_status check_shape(dynconv_shape s, bool need_c) {
    if (s.n <= 0 || s.h <= 0 || s.w <= 0) return DYNCONV_ERR_SHAPE;
    if (need_c && s.c <= 0) return DYNCONV_ERR_SHAPE;
    if (positions(s) > kMaxPositions) return DYNCONV_ERR_SHAPE;
    if (s.w > kMaxSeg * kWave) return DYNCONV_ERR_UNSUPPORTED;
    return DYNCONV_OK;
}

dynconv_status check_channels(int c) {
    if (c < 8 || c > kMaxC || c % 8 != 0) return DYNCONV_ERR_UNSUPPORTED;
    return DYNCONV_OK;
}

dynconv_status check_block(const dynconv_block *b, dynconv_shape s, bool need_mask) {
    if (!b) return DYNCONV_ERR_NULL;
    if (!b->w_expand || !b->b_expand || !b->w_dw || !b->b_dw || !b->w_project || !b->b_project)
        return DYNCONV_ERR_NULL;
    if (need_mask && !b->w_mask) return DYNCONV_ERR_NULL;
    if (b->c_in <= 0 || b->c_hidden <= 0 || b->c_out <= 0) return DYNCONV_ERR_SHAPE;
    if (b->c_in != s.c) return DYNCONV_ERR_SHAPE;
    if (b->c_out != b->c_in) return DYNCONV_ERR_UNSUPPORTED;  // identity path of Eq. 3
    if (dynconv_status st = check_channels(b->c_in)) return st;
    if (b->c_hidden < 16 || b->c_hidden > kMaxE || b->c_hidden % 16 != 0) return DYNCONV_ERR_UNSUPPORTED;
    for (int a : {b->act_expand, b->act_dw, b->act_project})
        if (a < DYNCONV_ACT_NONE || a > DYNCONV_ACT_RELU6) return DYNCONV_ERR_ARG;
    if (!aligned16(b->w_expand) || !aligned16(b->w_dw) || !aligned16(b->w_project) ||
        !aligned16(b->b_expand) || !aligned16(b->b_dw) || !aligned16(b->b_project))
        return DYNCONV_ERR_ALIGN;
    return DYNCONV_OK;
}

bool ranges_overlap(const void *a, size_t na, const void *b, size_t nb) {
    uintptr_t x0 = reinterpret_cast<uintptr_t>(a), y0 = reinterpret_cast<uintptr_t>(b);
    return x0 < y0 + nb && y0 < x0 + na;
}

dynconv_status launch_status() {
    return hipGetLastError() == hipSuccess ? DYNCONV_OK : DYNCONV_ERR_HIP;
}

// whole groups of 8 workgroups (one per XCD)
int grid_for_rows(int64_t rows) {
    int64_t tiles = (rows + 15) / 16;
    int64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks < 1) blocks = 1;
    if (blocks > kMaxGrid) blocks = kMaxGrid;
    return static_cast<int>((blocks + 7) / 8 * 8);
}

// Optional per-launch timing: launch i gets the event pair (ev[2i], ev[2i+1]),
// which the runtime stamps at the start and the end of that kernel.
struct Marks {
    hipEvent_t const *ev = nullptr;
    int32_t n = 0;  // number of events
    int32_t i = 0;  // launches so far
    void next(hipEvent_t *start, hipEvent_t *stop) {
        if (ev && 2 * i + 1 < n) {
            *start = ev[2 * i];
            *stop = ev[2 * i + 1];
        }
        ++i;
    }
};

template <typename... KArgs, typename... Args>
void launch(Marks &mk, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t st,
            Args... args) {
    hipEvent_t start = nullptr, stop = nullptr;
    mk.next(&start, &stop);
    hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(lds), st, start, stop, 0u,
                          static_cast<KArgs>(args)...);
}

// ------------------------------------------------------------ workspaces
struct IndexScratch {
    int2 *rowcnt;
    int2 *rowoff;
    uint64_t *words;  // mask words, [N*H][ceil(W/64)]
};

size_t index_scratch_bytes(dynconv_shape s) {
    int64_t rows = static_cast<int64_t>(s.n) * s.h;
    int64_t nseg = (s.w + kWave - 1) / kWave;
    return align_up(sizeof(int2) * rows) + align_up(sizeof(int2) * (rows + 1)) +
           align_up(sizeof(uint64_t) * rows * nseg);
}

IndexScratch carve_index_scratch(void *ws, dynconv_shape s) {
    int64_t rows = static_cast<int64_t>(s.n) * s.h;
    char *p = static_cast<char *>(ws);
    IndexScratch sc;
    sc.rowcnt = reinterpret_cast<int2 *>(p);
    p += align_up(sizeof(int2) * rows);
    sc.rowoff = reinterpret_cast<int2 *>(p);
    p += align_up(sizeof(int2) * (rows + 1));
    sc.words = reinterpret_cast<uint64_t *>(p);
    return sc;
}

// the expanded tensor: N*H*W rows plus one all-zero row for missing neighbours
size_t hidden_bytes(dynconv_shape s, int E, dynconv_dtype dt) {
    return align_up((static_cast<size_t>(positions(s)) + 1) * E * dtype_size(dt));
}

// base + off as an address.  The walks that only list launch names pass a
// null base and never dereference: integer arithmetic keeps that defined.
template <typename P = char>
P *at(const void *base, size_t off) {
    return reinterpret_cast<P *>(reinterpret_cast<uintptr_t>(base) + off);
}

// ------------------------------------------------------------ launches
template <typename T>
void launch_mask(const void *x, dynconv_shape s, const float *w_m, float b_m, uint8_t *mask,
                 float *logits, int mode, hipStream_t st, Marks &mk) {
    int64_t n = positions(s);
    int grid = static_cast<int>((n + kBlock - 1) / kBlock);
    launch(mk, k_mask<T>, dim3(grid), dim3(kBlock), 0, st, static_cast<const T *>(x), n, s.c, w_m,
           b_m, mask, logits, mode);
}

void launch_indices(const uint8_t *mask, dynconv_shape s, int dilate, const dynconv_indices *idx,
                    void *ws, hipStream_t st, Marks &mk) {
    IndexScratch sc = carve_index_scratch(ws, s);
    int64_t rows = static_cast<int64_t>(s.n) * s.h;
    int grid = static_cast<int>((rows + kWavesPerBlock - 1) / kWavesPerBlock);
    launch(mk, k_rowcount, dim3(grid), dim3(kBlock), 0, st, mask, s.n, s.h, s.w, dilate,
                       sc.rowcnt, sc.words);
    launch(mk, k_rowscan, dim3(1), dim3(kScanThreads), 0, st, sc.rowcnt, rows, sc.rowoff,
                       idx->counts);
    launch(mk, k_compact, dim3(grid), dim3(kBlock), 0, st, static_cast<const uint64_t *>(sc.words),
                       s.n, s.h, s.w, dilate, sc.rowoff, idx->active, idx->dilated, idx->nbr);
}

// expansion weights (rows of C+8) and bias staged in LDS when they fit in 64 KiB
constexpr size_t kMaxDynLds = 64 * 1024;
template <typename T>
size_t expand_lds_bytes(int C, int E) {
    return ((static_cast<size_t>(E) * (C + 8) * sizeof(T) + 15) & ~size_t(15)) + 4 * static_cast<size_t>(E);
}

template <typename T, bool DENSE, int MAXKS>
void launch_expand_k(const void *x, dynconv_shape s, const dynconv_block *b, const int32_t *dil,
                     const int32_t *counts, void *h1, hipStream_t st, Marks &mk) {
    int64_t rows = positions(s);
    // hidden-channel slabs whose expansion weights and biases fit in LDS
    int eslab = b->c_hidden;
    if (expand_lds_bytes<T>(b->c_in, eslab) > kMaxDynLds) {
        const size_t per_ch = (b->c_in + 8) * sizeof(T) + 4;
        eslab = static_cast<int>((kMaxDynLds - 16) / per_ch) / 16 * 16;
    }
    const int nslabs = (b->c_hidden + eslab - 1) / eslab;
    const int gps = grid_for_rows(rows);
    const size_t lds = expand_lds_bytes<T>(b->c_in, eslab);
    launch(mk, k_expand<T, DENSE, MAXKS, true>, dim3(gps * nslabs), dim3(kBlock), lds, st,
           static_cast<const T *>(x), b->c_in, b->c_hidden, static_cast<const T *>(b->w_expand),
           b->b_expand, b->act_expand, dil, counts, rows, static_cast<T *>(h1), eslab, gps);
}

template <typename T, bool DENSE>
void launch_expand(const void *x, dynconv_shape s, const dynconv_block *b, const int32_t *dil,
                   const int32_t *counts, void *h1, hipStream_t st, Marks &mk) {
    int ks = (b->c_in + 31) / 32;
    if (ks <= 1) launch_expand_k<T, DENSE, 1>(x, s, b, dil, counts, h1, st, mk);
    else if (ks <= 2) launch_expand_k<T, DENSE, 2>(x, s, b, dil, counts, h1, st, mk);
    else if (ks <= 4) launch_expand_k<T, DENSE, 4>(x, s, b, dil, counts, h1, st, mk);
    else launch_expand_k<T, DENSE, 8>(x, s, b, dil, counts, h1, st, mk);
}

template <typename T, bool DENSE, int MAXMT>
void launch_dw_project_k(const void *h1, const void *x, void *y, dynconv_shape s,
                         const dynconv_block *b, const int32_t *act, const int32_t *nbr,
                         const int32_t *counts, int nos, hipStream_t st, Marks &mk) {
    int64_t rows = positions(s);
    const int64_t groups = (rows + 16 * kDwGroup - 1) / (16 * kDwGroup);
    const int64_t g = groups < kMaxDwGrid ? (groups < 1 ? 1 : groups) : kMaxDwGrid;
    // whole groups of 8 (one per XCD), each slot with all its output slabs
    const int grid = static_cast<int>((g + 7) / 8 * 8 * nos);
    auto kern = nos > 1 ? k_dw_project<T, DENSE, MAXMT, true> : k_dw_project<T, DENSE, MAXMT, false>;
    launch(mk, kern, dim3(grid), dim3(kBlock), dw_lds_bytes<T>(),
                       st, static_cast<const T *>(h1), static_cast<const T *>(x), static_cast<T *>(y),
                       s.n, s.h, s.w, s.c, b->c_hidden, static_cast<const T *>(b->w_dw), b->b_dw,
                       b->act_dw, static_cast<const T *>(b->w_project), b->b_project, b->act_project,
                       act, nbr, counts, nos);
}

// Output slabs of the depthwise-projection: when the capacity has fewer than
// kDwTargetItems groups, the output tiles are cut into slabs of 2, 4 or 8
// tiles so that groups x slabs reaches that many work items (or one slab per
// tile pair).
constexpr int64_t kDwTargetItems = 512;

template <typename T, bool DENSE>
void launch_dw_project(const void *h1, const void *x, void *y, dynconv_shape s,
                       const dynconv_block *b, const int32_t *act, const int32_t *nbr,
                       const int32_t *counts, hipStream_t st, Marks &mk) {
    const int nmt = (b->c_out + 15) / 16;
    const int64_t groups = (positions(s) + 16 * kDwGroup - 1) / (16 * kDwGroup);
    int want = 1;
    if (groups < kDwTargetItems) {
        const int64_t w = (kDwTargetItems + groups - 1) / (groups < 1 ? 1 : groups);
        want = static_cast<int>(w < nmt ? w : nmt);
    }
    const int per = (nmt + want - 1) / want;  // tiles per slab before rounding to an instantiation
    const int tiles = per <= 2 ? 2 : per <= 4 ? 4 : per <= 8 ? 8 : 16;
    const int nos = (nmt + tiles - 1) / tiles;
    if (tiles == 2) launch_dw_project_k<T, DENSE, 2>(h1, x, y, s, b, act, nbr, counts, nos, st, mk);
    else if (tiles == 4) launch_dw_project_k<T, DENSE, 4>(h1, x, y, s, b, act, nbr, counts, nos, st, mk);
    else if (tiles == 8) launch_dw_project_k<T, DENSE, 8>(h1, x, y, s, b, act, nbr, counts, nos, st, mk);
    else launch_dw_project_k<T, DENSE, 16>(h1, x, y, s, b, act, nbr, counts, nos, st, mk);
}

template <typename T>
void launch_block(const void *x, void *y, dynconv_shape s, const dynconv_block *b,
                  const dynconv_indices *idx, void *h1, hipStream_t st, Marks &mk) {
    if (idx) {
        launch_expand<T, false>(x, s, b, idx->dilated, idx->counts, h1, st, mk);
        launch_dw_project<T, false>(h1, x, y, s, b, idx->active, idx->nbr, idx->counts, st, mk);
    } else {
        launch_expand<T, true>(x, s, b, nullptr, nullptr, h1, st, mk);
        launch_dw_project<T, true>(h1, x, y, s, b, nullptr, nullptr, nullptr, st, mk);
    }
}

void launch_copy(const void *src, void *dst, size_t bytes, hipStream_t st, Marks &mk) {
    int64_t n16 = static_cast<int64_t>(bytes / 16);
    int64_t blocks = (n16 + kBlock - 1) / kBlock;
    int grid = static_cast<int>(blocks < 4096 ? (blocks < 1 ? 1 : blocks) : 4096);
    launch(mk, k_copy16, dim3(grid), dim3(kBlock), 0, st, static_cast<const uint4 *>(src),
           static_cast<uint4 *>(dst), n16);
}

void dispatch_mask(dynconv_dtype dt, const void *x, dynconv_shape s, const float *w_m, float b_m,
                   uint8_t *mask, float *logits, int mode, hipStream_t st, Marks &mk) {
    if (dt == DYNCONV_F32) launch_mask<float>(x, s, w_m, b_m, mask, logits, mode, st, mk);
    else if (dt == DYNCONV_F16) launch_mask<half_t>(x, s, w_m, b_m, mask, logits, mode, st, mk);
    else launch_mask<bf16_t>(x, s, w_m, b_m, mask, logits, mode, st, mk);
}

// ------------------------------------------------------------ fused block
// Patches of the one-launch block kernel: the configuration PatchCfgOf picks
// for the element type and channel bound.
template <typename T, int MAXC>
PatchGeom fused_geom_t(dynconv_shape s) {
    typedef typename PatchCfgOf<T, MAXC>::type CFG;
    return patch_geom(s.n, s.h, s.w, CFG::kOwn, CFG::kRegion);
}

PatchGeom fused_geom(dynconv_shape s, dynconv_dtype dt) {
    if (dt == DYNCONV_F32) return s.c <= 32 ? fused_geom_t<float, 32>(s) : fused_geom_t<float, 64>(s);
    if (s.c <= 32) return fused_geom_t<half_t, 32>(s);
    return s.c <= 64 ? fused_geom_t<half_t, 64>(s) : fused_geom_t<half_t, 128>(s);
}

int fused_patch_count(dynconv_shape s, dynconv_dtype dt) {
    const PatchGeom p = fused_geom(s, dt);
    return s.n * p.nph * p.npw;
}

// Per-launch mask plumbing of one fused block: where its mask comes from
// (mask_in, or computed in the kernel with the block's own mask unit and
// written to mask_self), where the next block's mask goes, and where the
// patches' active and dilated counts go.
struct FusedMasks {
    const uint8_t *mask_in = nullptr;
    bool self = false;
    uint8_t *mask_self = nullptr;
    uint8_t *mask_next = nullptr;
    int32_t *band_counts = nullptr;
    // nonzero: the block is the branch of a ShuffleNetV2 unit with this many
    // channels per half, reading and writing the unit's full rows
    int shuffle_cb = 0;
    int mask_mode = 0;  // hard decision of the mask units (mask_decision)
};

template <typename T, bool DENSE, int MAXKS, int MAXMT, int MAXC>
void launch_fused_k(const void *src, void *dst, dynconv_shape s, const dynconv_block *b,
                    const dynconv_block *next, const FusedMasks &fm, hipStream_t st, Marks &mk) {
    typedef typename PatchCfgOf<T, MAXC>::type CFG;
    const PatchGeom p = fused_geom_t<T, MAXC>(s);
    const int npatch = s.n * p.nph * p.npw;
    const int grid = (npatch + 7) / 8 * 8;  // whole groups of 8 (one per XCD)
    auto kern = fm.shuffle_cb ? k_block_fused<T, DENSE, MAXKS, MAXMT, MAXC, CFG, true>
                              : k_block_fused<T, DENSE, MAXKS, MAXMT, MAXC, CFG, false>;
    launch(mk, kern, dim3(grid), dim3(CFG::kThreads), 0, st,
           static_cast<const T *>(src), static_cast<T *>(dst), s.n, s.h, s.w, s.c, b->c_hidden, p.R, p.Wu,
           fm.shuffle_cb, fm.mask_in, fm.self ? b->w_mask : nullptr, b->b_mask, fm.mask_self,
           static_cast<const T *>(b->w_expand), b->b_expand, b->act_expand,
           static_cast<const T *>(b->w_dw), b->b_dw, b->act_dw,
           static_cast<const T *>(b->w_project), b->b_project, b->act_project,
           next ? next->w_mask : nullptr, next ? next->b_mask : 0.0f,
           next ? fm.mask_next : nullptr, fm.band_counts, fm.mask_mode);
}

template <typename T, bool DENSE>
void launch_fused(const void *src, void *dst, dynconv_shape s, const dynconv_block *b,
                  const dynconv_block *next, const FusedMasks &fm, hipStream_t st, Marks &mk) {
    if (s.c <= 32)
        launch_fused_k<T, DENSE, 1, 2, 32>(src, dst, s, b, next, fm, st, mk);
    else if (s.c <= 64)
        launch_fused_k<T, DENSE, 2, 4, 64>(src, dst, s, b, next, fm, st, mk);
    else if constexpr (sizeof(T) == 2)  // 16-bit only (use_fused keeps fp32 at 64)
        launch_fused_k<T, DENSE, 4, 8, 128>(src, dst, s, b, next, fm, st, mk);
}

void dispatch_fused(dynconv_dtype dt, bool dense, const void *src, void *dst, dynconv_shape s,
                    const dynconv_block *b, const dynconv_block *next, const FusedMasks &fm,
                    hipStream_t st, Marks &mk) {
#define DC_FUSED(T)                                                                  \
    (dense ? launch_fused<T, true>(src, dst, s, b, nullptr, dense_fm, st, mk)        \
           : launch_fused<T, false>(src, dst, s, b, next, fm, st, mk))
    FusedMasks dense_fm;
    dense_fm.shuffle_cb = fm.shuffle_cb;
    if (dt == DYNCONV_F32) DC_FUSED(float);
    else if (dt == DYNCONV_F16) DC_FUSED(half_t);
    else DC_FUSED(bf16_t);
#undef DC_FUSED
}

// ------------------------------------------------------------ balanced cells
// Compute units of the current device (the persistent grid of k_block_cells).
int device_cus() {
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cached[dev].load(std::memory_order_relaxed);
    if (v <= 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
            v = 256;
        cached[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

int64_t cell_count(dynconv_shape s) { return static_cast<int64_t>(s.n) * cells_per_image(s.h, s.w); }

// Persistent grid: at most one workgroup per CU, at least one cell per wave.
int cells_shares(dynconv_shape s) {
    const int64_t by_cells = (cell_count(s) + kCellWaves - 1) / kCellWaves;
    return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(device_cus(), by_cells)));
}

template <typename T>
void launch_mask_cells(const void *x, dynconv_shape s, const dynconv_block *b, uint8_t *mask, uint8_t *cnt,
                       int mode, hipStream_t st, Marks &mk) {
    const int64_t per_group = static_cast<int64_t>(kCellsPerMaskWave) * kWavesPerBlock;
    const int64_t grid = (cell_count(s) + per_group - 1) / per_group;
    launch(mk, k_mask_cells<T>, dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, st, static_cast<const T *>(x),
           s.n, s.h, s.w, s.c, b->w_mask, b->b_mask, mask, cnt, mode);
}

struct CellMasks {
    const uint8_t *mask_in = nullptr, *cnt_in = nullptr;
    uint8_t *mask_next = nullptr, *cnt_next = nullptr;
    int32_t *band_counts = nullptr;
    int mask_mode = 0;
};

template <typename T, bool DENSE>
void launch_cells(const void *src, void *dst, dynconv_shape s, const dynconv_block *b, const dynconv_block *next,
                  const CellMasks &cm, hipStream_t st, Marks &mk) {
    const int G = cells_shares(s);
    const int grid = (G + 7) / 8 * 8;
    launch(mk, k_block_cells<T, DENSE>, dim3(grid), dim3(kCellThreads), 0, st, static_cast<const T *>(src),
           static_cast<T *>(dst), s.n, s.h, s.w, s.c, b->c_hidden, G, cm.mask_in, cm.cnt_in,
           static_cast<const T *>(b->w_expand), b->b_expand, b->act_expand,
           static_cast<const T *>(b->w_dw), b->b_dw, b->act_dw,
           static_cast<const T *>(b->w_project), b->b_project, b->act_project,
           next ? next->w_mask : nullptr, next ? next->b_mask : 0.0f, next ? cm.mask_next : nullptr,
           next ? cm.cnt_next : nullptr, cm.band_counts, cm.mask_mode);
}

void dispatch_cells(dynconv_dtype dt, bool dense, const void *src, void *dst, dynconv_shape s,
                    const dynconv_block *b, const dynconv_block *next, const CellMasks &cm, hipStream_t st,
                    Marks &mk) {
    if (dt == DYNCONV_F16) {
        if (dense) launch_cells<half_t, true>(src, dst, s, b, nullptr, cm, st, mk);
        else launch_cells<half_t, false>(src, dst, s, b, next, cm, st, mk);
    } else {
        if (dense) launch_cells<bf16_t, true>(src, dst, s, b, nullptr, cm, st, mk);
        else launch_cells<bf16_t, false>(src, dst, s, b, next, cm, st, mk);
    }
}

void dispatch_mask_cells(dynconv_dtype dt, const void *x, dynconv_shape s, const dynconv_block *b, uint8_t *mask,
                         uint8_t *cnt, int mode, hipStream_t st, Marks &mk) {
    if (dt == DYNCONV_F16) launch_mask_cells<half_t>(x, s, b, mask, cnt, mode, st, mk);
    else launch_mask_cells<bf16_t>(x, s, b, mask, cnt, mode, st, mk);
}

void dispatch_block(dynconv_dtype dt, const void *x, void *y, dynconv_shape s, const dynconv_block *b,
                    const dynconv_indices *idx, void *h1, hipStream_t st, Marks &mk) {
    if (dt == DYNCONV_F32) launch_block<float>(x, y, s, b, idx, h1, st, mk);
    else if (dt == DYNCONV_F16) launch_block<half_t>(x, y, s, b, idx, h1, st, mk);
    else launch_block<bf16_t>(x, y, s, b, idx, h1, st, mk);
}

// ------------------------------------------------------------ stacks
constexpr int32_t kStackDense = 1;
constexpr int32_t kStackUnfused = 2;
constexpr int32_t kStackGSoftmax = 4;
constexpr int32_t kStackFlags = kStackDense | kStackUnfused | kStackGSoftmax;

int mask_mode_of(int32_t flags) { return (flags & kStackGSoftmax) ? 1 : 0; }

// The one-launch block kernel covers up to 64 channels in fp32 and 128 in
// fp16/bf16; wider blocks run the unfused kernel chain.
bool use_fused(dynconv_shape s, dynconv_dtype dt, int32_t flags) {
    return !(flags & kStackUnfused) && s.c <= (dt == DYNCONV_F32 ? kMaxFusedC : kMaxFusedC16);
}

// Narrow 16-bit blocks (at most 32 channels, 192 hidden) run the
// work-balanced cell kernel, which keeps all weights of a block in LDS.
bool use_cells(dynconv_shape s, dynconv_dtype dt, const dynconv_block *blks, int32_t n_blocks, int32_t flags) {
    if ((flags & kStackUnfused) || dt == DYNCONV_F32 || s.c > kCellMaxC) return false;
    // the kernel's share bounds (cell count x workgroup count) are 32-bit
    if (cell_count(s) * cells_shares(s) > 0xffffffffLL) return false;
    for (int32_t b = 0; b < n_blocks; ++b)
        if (blks[b].c_hidden > kCellMaxE) return false;
    return true;
}

struct StackLayout {
    bool fused, cells;
    size_t masks, mask2, tbuf, active, dilated, nbr, counts, bands, scratch, hidden, cc0, cc1, total;
};

// allow_cells: the ShuffleNetV2 units run their branch on the patch kernel
// (its staging reads the unit's rows directly), never on the cell kernel.
StackLayout stack_layout(dynconv_shape s, const dynconv_block *blks, int32_t n_blocks,
                         dynconv_dtype dt, int32_t flags, bool allow_cells = true) {
    StackLayout L{};
    L.fused = use_fused(s, dt, flags);
    L.cells = allow_cells && L.fused && use_cells(s, dt, blks, n_blocks, flags);
    size_t npos = static_cast<size_t>(positions(s));
    size_t off = 0;
    if (L.cells) {
        const size_t ncells = static_cast<size_t>(cell_count(s));
        L.tbuf = off;   off += align_up(npos * s.c * dtype_size(dt));
        L.masks = off;  off += align_up(npos);
        L.mask2 = off;  off += align_up(npos);
        L.counts = off; off += align_up(8 * static_cast<size_t>(n_blocks));
        L.bands = off;  off += align_up(8 * static_cast<size_t>(n_blocks) * ncells);
        L.cc0 = off;    off += align_up(ncells);
        L.cc1 = off;    off += align_up(ncells);
    } else if (L.fused) {
        L.tbuf = off;   off += align_up(npos * s.c * dtype_size(dt));
        L.masks = off;  off += align_up(npos);
        L.mask2 = off;  off += align_up(npos);
        L.counts = off; off += align_up(8 * static_cast<size_t>(n_blocks));
        L.bands = off;  off += align_up(8 * static_cast<size_t>(n_blocks) * fused_patch_count(s, dt));
    } else {
        int emax = 0;
        for (int32_t b = 0; b < n_blocks; ++b)
            if (blks[b].c_hidden > emax) emax = blks[b].c_hidden;
        L.masks = off;   off += align_up(npos);
        L.active = off;  off += align_up(4 * npos);
        L.dilated = off; off += align_up(4 * npos);
        L.nbr = off;     off += align_up(36 * npos);
        L.counts = off;  off += align_up(8 * static_cast<size_t>(n_blocks));
        L.scratch = off; off += index_scratch_bytes(s);
        L.hidden = off;  off += hidden_bytes(s, emax, dt);
    }
    L.total = off;
    return L;
}

dynconv_status stack_checked(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                             const dynconv_block *blks, int32_t n_blocks, int32_t flags) {
    if (!x || !y || !blks) return DYNCONV_ERR_NULL;
    if (!dtype_ok(dt)) return DYNCONV_ERR_DTYPE;
    if (n_blocks < 1 || n_blocks > kMaxBlocks) return DYNCONV_ERR_ARG;
    if (flags & ~kStackFlags) return DYNCONV_ERR_ARG;
    if (dynconv_status st = check_shape(s, true)) return st;
    for (int32_t b = 0; b < n_blocks; ++b)
        if (dynconv_status st = check_block(&blks[b], s, !(flags & kStackDense))) return st;
    if (!aligned16(x) || !aligned16(y)) return DYNCONV_ERR_ALIGN;
    size_t bytes = static_cast<size_t>(positions(s)) * s.c * dtype_size(dt);
    if (x != y && ranges_overlap(x, bytes, y, bytes)) return DYNCONV_ERR_SHAPE;
    return DYNCONV_OK;
}

// Walks the launch sequence of a stack.  With exec == false it only records
// the kernel names (what dynconv_stack_launch_names reports).
struct Plan {
    bool exec;
    const char **names;
    int32_t cap;
    int32_t count = 0;
    bool list_counts = true;  // a plan without execution lists the count reduction
    bool note(const char *name) {
        if (names && count < cap) names[count] = name;
        ++count;
        return exec;
    }
};

void stack_walk(const void *x, void *y, dynconv_shape s, dynconv_dtype dt, const dynconv_block *blks,
                int32_t n_blocks, int32_t flags, uint8_t *masks, int32_t *counts, char *base,
                const StackLayout &L, hipStream_t st, Marks &mk, Plan &plan, bool in_place) {
    const bool dense = flags & kStackDense;
    const size_t npos = static_cast<size_t>(positions(s));
    const size_t bytes = npos * s.c * dtype_size(dt);
    int32_t *cnt_all = counts ? counts : at<int32_t>(base, L.counts);
    if (L.cells) {
        // Ping-pong between y and a scratch copy so that the last block writes y.
        void *tb = at(base, L.tbuf);
        const void *src = x;
        if (in_place && (n_blocks % 2 == 1)) {
            if (plan.note("k_copy16")) launch_copy(x, tb, bytes, st, mk);  // keeps y free for block 0
            src = tb;
        }
        auto mask_of = [&](int32_t b) -> uint8_t * {
            if (masks) return masks + static_cast<size_t>(b) * npos;
            return at<uint8_t>(base, ((b % 2) ? L.mask2 : L.masks));
        };
        auto cnt_of = [&](int32_t b) -> uint8_t * {
            return at<uint8_t>(base, ((b % 2) ? L.cc1 : L.cc0));
        };
        const int64_t ncells = cell_count(s);
        int32_t *band_counts = at<int32_t>(base, L.bands);
        // the first block's mask unit and its per-cell active counts
        if (!dense && plan.note("k_mask_cells"))
            dispatch_mask_cells(dt, src, s, &blks[0], mask_of(0), cnt_of(0), mask_mode_of(flags), st, mk);
        for (int32_t b = 0; b < n_blocks; ++b) {
            void *dst = ((n_blocks - 1 - b) % 2 == 0) ? y : tb;
            const dynconv_block *next = (b + 1 < n_blocks) ? &blks[b + 1] : nullptr;
            CellMasks cm;
            cm.mask_mode = mask_mode_of(flags);
            cm.mask_in = mask_of(b);
            cm.cnt_in = cnt_of(b);
            cm.mask_next = next ? mask_of(b + 1) : nullptr;
            cm.cnt_next = next ? cnt_of(b + 1) : nullptr;
            cm.band_counts = counts ? band_counts + static_cast<size_t>(2) * ncells * b : nullptr;
            if (plan.note("k_block_cells")) dispatch_cells(dt, dense, src, dst, s, &blks[b], next, cm, st, mk);
            src = dst;
        }
        if (!dense && (counts || (!plan.exec && plan.list_counts)) && plan.note("k_band_counts"))
            launch(mk, k_band_counts, dim3(n_blocks), dim3(kBlock), 0, st,
                   static_cast<const int32_t *>(band_counts), static_cast<int>(ncells), cnt_all);
        return;
    }
    if (L.fused) {
        // Ping-pong between y and a scratch copy so that the last block writes y.
        void *tb = at(base, L.tbuf);
        const void *src = x;
        if (in_place && (n_blocks % 2 == 1)) {
            if (plan.note("k_copy16")) launch_copy(x, tb, bytes, st, mk);  // keeps y free for block 0
            src = tb;
        }
        auto mask_of = [&](int32_t b) -> uint8_t * {
            if (masks) return masks + static_cast<size_t>(b) * npos;
            return at<uint8_t>(base, ((b % 2) ? L.mask2 : L.masks));
        };
        const int nbands = fused_patch_count(s, dt);
        int32_t *band_counts = at<int32_t>(base, L.bands);
        for (int32_t b = 0; b < n_blocks; ++b) {
            void *dst = ((n_blocks - 1 - b) % 2 == 0) ? y : tb;
            const dynconv_block *next = (b + 1 < n_blocks) ? &blks[b + 1] : nullptr;
            FusedMasks fm;
            fm.mask_mode = mask_mode_of(flags);
            fm.self = (b == 0);  // block 0 runs its own mask unit on the staged x
            fm.mask_in = (b == 0) ? nullptr : mask_of(b);
            fm.mask_self = mask_of(0);
            fm.mask_next = next ? mask_of(b + 1) : nullptr;
            fm.band_counts = band_counts + static_cast<size_t>(2) * nbands * b;
            if (plan.note("k_block_fused")) dispatch_fused(dt, dense, src, dst, s, &blks[b], next, fm, st, mk);
            src = dst;
        }
        // P, P_d per block only on request (listed in every plan)
        if (!dense && (counts || (!plan.exec && plan.list_counts)) && plan.note("k_band_counts"))
            launch(mk, k_band_counts, dim3(n_blocks), dim3(kBlock), 0, st,
                   static_cast<const int32_t *>(band_counts), nbands, cnt_all);
        return;
    }
    // Unfused chain, in place on y.
    if (!in_place && plan.note("k_copy16")) launch_copy(x, y, bytes, st, mk);
    void *h1 = at(base, L.hidden);
    if (dense) {
        for (int32_t b = 0; b < n_blocks; ++b) {
            bool run = plan.note("k_expand");
            plan.note("k_dw_project");
            if (run) dispatch_block(dt, y, y, s, &blks[b], nullptr, h1, st, mk);
        }
        return;
    }
    dynconv_indices idx;
    idx.active = at<int32_t>(base, L.active);
    idx.dilated = at<int32_t>(base, L.dilated);
    idx.nbr = at<int32_t>(base, L.nbr);
    idx.capacity = static_cast<int64_t>(npos);
    void *scratch = at(base, L.scratch);
    for (int32_t b = 0; b < n_blocks; ++b) {
        uint8_t *mask_b = masks ? masks + static_cast<size_t>(b) * npos
                                : at<uint8_t>(base, L.masks);
        idx.counts = cnt_all + 2 * b;
        bool run = plan.note("k_mask");
        plan.note("k_rowcount");
        plan.note("k_rowscan");
        plan.note("k_compact");
        plan.note("k_expand");
        plan.note("k_dw_project");
        if (run) {
            dispatch_mask(dt, y, s, blks[b].w_mask, blks[b].b_mask, mask_b, nullptr, mask_mode_of(flags), st, mk);
            launch_indices(mask_b, s, 1, &idx, scratch, st, mk);
            dispatch_block(dt, y, y, s, &blks[b], &idx, h1, st, mk);
        }
    }
}

// ------------------------------------------------------------ ShuffleNetV2 units
// Unit outputs alternate between y and a full-row scratch buffer so that the
// last unit writes y.  When the branch takes the one-launch block and a half
// row is whole 4-byte words, that kernel reads the branch half of the unit's
// input rows and writes the shuffled output rows itself (one launch per
// unit).  Otherwise the branch runs on compact cp-channel rows (x2
// zero-extended, cp = the branch block's c_in), filled by k_shuffle_split /
// k_shuffle_merge; two such buffers alternate.
struct ShuffleLayout {
    bool direct;
    size_t xa, xb, full, inner, total;
    StackLayout in;
};

bool shuffle_direct(dynconv_shape s, const dynconv_block *br, dynconv_dtype dt, int32_t flags) {
    dynconv_shape bs = s;
    bs.c = br[0].c_in;
    return use_fused(bs, dt, flags) && (s.c / 2) * dtype_size(dt) % 4 == 0;
}

dynconv_shape branch_shape(dynconv_shape s, const dynconv_block *br) {
    dynconv_shape b = s;
    b.c = br[0].c_in;
    return b;
}

ShuffleLayout shuffle_layout(dynconv_shape s, const dynconv_block *br, int32_t n_units, dynconv_dtype dt,
                             int32_t flags) {
    const dynconv_shape bs = branch_shape(s, br);
    const size_t npos = static_cast<size_t>(positions(s));
    ShuffleLayout L{};
    L.direct = shuffle_direct(s, br, dt, flags);
    const size_t rows = L.direct ? 0 : align_up(npos * bs.c * dtype_size(dt));
    size_t off = 0;
    L.xa = off;    off += rows;
    L.xb = off;    off += rows;
    L.full = off;  off += (n_units > 1) ? align_up(npos * s.c * dtype_size(dt)) : 0;
    L.inner = off;
    L.in = stack_layout(bs, br, n_units, dt, flags, false);
    off += L.in.total;
    L.total = off;
    return L;
}

dynconv_status shuffle_checked(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                               const dynconv_block *br, int32_t n_units, int32_t flags) {
    if (!x || !y || !br) return DYNCONV_ERR_NULL;
    if (!dtype_ok(dt)) return DYNCONV_ERR_DTYPE;
    if (n_units < 1 || n_units > kMaxBlocks) return DYNCONV_ERR_ARG;
    if (flags & ~kStackFlags) return DYNCONV_ERR_ARG;
    if (dynconv_status st = check_shape(s, true)) return st;
    if (s.c % 2 != 0) return DYNCONV_ERR_SHAPE;
    const dynconv_shape bs = branch_shape(s, br);
    if (bs.c < s.c / 2) return DYNCONV_ERR_SHAPE;
    for (int32_t u = 0; u < n_units; ++u)
        if (dynconv_status st = check_block(&br[u], bs, !(flags & kStackDense))) return st;
    if (!aligned16(x) || !aligned16(y)) return DYNCONV_ERR_ALIGN;
    const size_t bytes = static_cast<size_t>(positions(s)) * s.c * dtype_size(dt);
    if (ranges_overlap(x, bytes, y, bytes)) return DYNCONV_ERR_SHAPE;
    return DYNCONV_OK;
}

int shuffle_grid(int64_t npos) {
    int64_t g = (npos + kShufRows - 1) / kShufRows;
    if (g > 8192) g = 8192;
    return static_cast<int>((g + 7) / 8 * 8);
}

void dispatch_split(dynconv_dtype dt, const void *x, void *xa, int64_t npos, int cb, int cp,
                    hipStream_t st, Marks &mk) {
#define DC_SPLIT(T)                                                                            \
    launch(mk, k_shuffle_split<T>, dim3(shuffle_grid(npos)), dim3(kBlock), 0, st,             \
           static_cast<const T *>(x), static_cast<T *>(xa), npos, cb, cp)
    if (dt == DYNCONV_F32) DC_SPLIT(float);
    else if (dt == DYNCONV_F16) DC_SPLIT(half_t);
    else DC_SPLIT(bf16_t);
#undef DC_SPLIT
}

void dispatch_merge(dynconv_dtype dt, const void *x, const void *br, void *y, void *xa, int64_t npos,
                    int cb, int cp, hipStream_t st, Marks &mk) {
#define DC_MERGE(T)                                                                            \
    launch(mk, k_shuffle_merge<T>, dim3(shuffle_grid(npos)), dim3(kBlock), 0, st,             \
           static_cast<const T *>(x), static_cast<const T *>(br), static_cast<T *>(y),       \
           static_cast<T *>(xa), npos, cb, cp)
    if (dt == DYNCONV_F32) DC_MERGE(float);
    else if (dt == DYNCONV_F16) DC_MERGE(half_t);
    else DC_MERGE(bf16_t);
#undef DC_MERGE
}

void shuffle_walk(const void *x, void *y, dynconv_shape s, dynconv_dtype dt, const dynconv_block *br,
                  int32_t n_units, int32_t flags, uint8_t *masks, int32_t *counts, char *base,
                  const ShuffleLayout &SL, hipStream_t st, Marks &mk, Plan &plan) {
    const bool dense = flags & kStackDense;
    const dynconv_shape bs = branch_shape(s, br);
    const int cb = s.c / 2, cp = bs.c;
    const int64_t npos = positions(s);
    const StackLayout &L = SL.in;
    char *ib = at(base, SL.inner);
    void *bufs[2] = {at(base, SL.xa), at(base, SL.xb)};
    void *full = at(base, SL.full);
    int32_t *cnt_all = counts ? counts : at<int32_t>(ib, L.counts);
    auto mask_of = [&](int32_t u) -> uint8_t * {
        if (masks) return masks + static_cast<size_t>(u) * npos;
        return at<uint8_t>(ib, L.masks);
    };
    auto out_of = [&](int32_t u) -> void * { return ((n_units - 1 - u) % 2 == 0) ? y : full; };
    // branch input of unit u: bufs[0] for the one-launch block (its output
    // goes to bufs[1]); bufs[u % 2] for the kernel chain, which runs in place
    auto in_of = [&](int32_t u) -> void * { return L.fused ? bufs[0] : bufs[u % 2]; };

    const int nbands = L.fused ? fused_patch_count(bs, dt) : 0;
    int32_t *band_counts = at<int32_t>(ib, L.bands);
    if (SL.direct) {
        for (int32_t u = 0; u < n_units; ++u) {
            FusedMasks fm;
            fm.mask_mode = mask_mode_of(flags);
            fm.shuffle_cb = cb;
            if (!dense) {
                fm.self = true;  // the unit's mask unit on the staged branch half
                fm.mask_self = masks ? mask_of(u) : nullptr;
                fm.band_counts = band_counts + static_cast<size_t>(2) * nbands * u;
            }
            const void *xu = (u == 0) ? x : out_of(u - 1);
            if (plan.note("k_block_fused")) dispatch_fused(dt, dense, xu, out_of(u), bs, &br[u], nullptr, fm, st, mk);
        }
        if (!dense && (counts || (!plan.exec && plan.list_counts)) && plan.note("k_band_counts"))
            launch(mk, k_band_counts, dim3(n_units), dim3(kBlock), 0, st,
                   static_cast<const int32_t *>(band_counts), nbands, cnt_all);
        return;
    }
    if (plan.note("k_shuffle_split")) dispatch_split(dt, x, in_of(0), npos, cb, cp, st, mk);
    dynconv_indices idx;
    idx.active = at<int32_t>(ib, L.active);
    idx.dilated = at<int32_t>(ib, L.dilated);
    idx.nbr = at<int32_t>(ib, L.nbr);
    idx.capacity = npos;
    for (int32_t u = 0; u < n_units; ++u) {
        const void *xu = (u == 0) ? x : out_of(u - 1);
        void *bin = in_of(u);
        const void *bout = bin;
        if (L.fused) {
            FusedMasks fm;
            fm.mask_mode = mask_mode_of(flags);
            if (!dense) {
                fm.self = true;  // the unit's mask unit on the staged branch input
                fm.mask_self = masks ? mask_of(u) : nullptr;
                fm.band_counts = band_counts + static_cast<size_t>(2) * nbands * u;
            }
            bout = bufs[1];
            if (plan.note("k_block_fused"))
                dispatch_fused(dt, dense, bin, bufs[1], bs, &br[u], nullptr, fm, st, mk);
        } else if (dense) {
            bool run = plan.note("k_expand");
            plan.note("k_dw_project");
            if (run) dispatch_block(dt, bin, bin, bs, &br[u], nullptr, at(ib, L.hidden), st, mk);
        } else {
            idx.counts = cnt_all + 2 * u;
            bool run = plan.note("k_mask");
            plan.note("k_rowcount");
            plan.note("k_rowscan");
            plan.note("k_compact");
            plan.note("k_expand");
            plan.note("k_dw_project");
            if (run) {
                dispatch_mask(dt, bin, bs, br[u].w_mask, br[u].b_mask, mask_of(u), nullptr, mask_mode_of(flags),
                              st, mk);
                launch_indices(mask_of(u), bs, 1, &idx, at(ib, L.scratch), st, mk);
                dispatch_block(dt, bin, bin, bs, &br[u], &idx, at(ib, L.hidden), st, mk);
            }
        }
        void *next_in = (u + 1 < n_units) ? in_of(u + 1) : nullptr;
        if (plan.note("k_shuffle_merge")) dispatch_merge(dt, xu, bout, out_of(u), next_in, npos, cb, cp, st, mk);
    }
    if (L.fused && !dense && (counts || (!plan.exec && plan.list_counts)) && plan.note("k_band_counts"))
        launch(mk, k_band_counts, dim3(n_units), dim3(kBlock), 0, st,
               static_cast<const int32_t *>(band_counts), nbands, cnt_all);
}

// ------------------------------------------------------------ whole networks
// A layer list (dynconv_layer) run on one stream: dense layers with the
// kernels of dense.h, gated blocks as one-block stacks.  Activations
// alternate between two buffers sized for the largest layer output; the
// last layer writes y.  Dense blocks keep their expanded tensor (H1, input
// resolution) and depthwise output (H2, output resolution) in two more
// buffers.
constexpr int kMaxLayers = 1024;

struct LayerShapes {
    dynconv_shape in, out;
    int hidden;  // dense blocks: hidden width
};

dynconv_status layer_shape(const dynconv_layer &L, dynconv_shape in, LayerShapes &o, bool need_mask) {
    o.in = in;
    o.out = in;
    o.hidden = 0;
    if (L.kind == DYNCONV_LAYER_CONV3X3) {
        if (!L.w || !L.b) return DYNCONV_ERR_NULL;
        if (L.c_in != in.c || L.c_in < 1 || L.c_in > 16) return DYNCONV_ERR_SHAPE;
        if (L.stride != 1 && L.stride != 2) return DYNCONV_ERR_ARG;
        if (L.c_out < 8 || L.c_out > 256 || L.c_out % 8) return DYNCONV_ERR_UNSUPPORTED;
        if (9 * L.c_in * L.c_out + L.c_out > 16384) return DYNCONV_ERR_UNSUPPORTED;  // fp32 weights in 64 KB of LDS
        if (L.act < DYNCONV_ACT_NONE || L.act > DYNCONV_ACT_RELU6) return DYNCONV_ERR_ARG;
        o.out.h = (in.h - 1) / L.stride + 1;
        o.out.w = (in.w - 1) / L.stride + 1;
        o.out.c = L.c_out;
        return DYNCONV_OK;
    }
    if (L.kind == DYNCONV_LAYER_CONV1X1) {
        if (!L.w || !L.b) return DYNCONV_ERR_NULL;
        if (L.c_in != in.c) return DYNCONV_ERR_SHAPE;
        if (L.c_in < 8 || L.c_in % 8 || L.c_out < 8 || L.c_out % 8 || L.c_out > 4096)
            return DYNCONV_ERR_UNSUPPORTED;
        if (L.act < DYNCONV_ACT_NONE || L.act > DYNCONV_ACT_RELU6) return DYNCONV_ERR_ARG;
        if (!aligned16(L.w)) return DYNCONV_ERR_ALIGN;
        o.out.c = L.c_out;
        return DYNCONV_OK;
    }
    if (L.kind != DYNCONV_LAYER_BLOCK) return DYNCONV_ERR_ARG;
    const dynconv_block &b = L.blk;
    if (L.stride != 1 && L.stride != 2) return DYNCONV_ERR_ARG;
    if (b.c_in != in.c) return DYNCONV_ERR_SHAPE;
    if (L.gated) {
        if (L.stride != 1 || b.c_out != b.c_in) return DYNCONV_ERR_UNSUPPORTED;
        if (dynconv_status st = check_block(&b, in, need_mask)) return st;
        if (!b.w_expand) return DYNCONV_ERR_NULL;
        return DYNCONV_OK;
    }
    if (!b.w_dw || !b.b_dw || !b.w_project || !b.b_project) return DYNCONV_ERR_NULL;
    if (b.w_expand && !b.b_expand) return DYNCONV_ERR_NULL;
    const int E = b.w_expand ? b.c_hidden : b.c_in;
    if (!b.w_expand && b.c_hidden != b.c_in) return DYNCONV_ERR_SHAPE;
    if (b.c_in % 8 || b.c_out % 8 || E % 8 || b.c_in < 8 || b.c_out < 8 || E > 1792 || b.c_out > 4096)
        return DYNCONV_ERR_UNSUPPORTED;
    for (int a : {b.act_expand, b.act_dw, b.act_project})
        if (a < DYNCONV_ACT_NONE || a > DYNCONV_ACT_RELU6) return DYNCONV_ERR_ARG;
    if ((b.w_expand && !aligned16(b.w_expand)) || !aligned16(b.w_project)) return DYNCONV_ERR_ALIGN;
    o.out.h = (in.h - 1) / L.stride + 1;
    o.out.w = (in.w - 1) / L.stride + 1;
    o.out.c = b.c_out;
    o.hidden = E;
    return DYNCONV_OK;
}

struct NetLayout {
    size_t act0, act1, h1, h2, masks, counts, inner, total;
    size_t act_bytes, inner_bytes;
    int ngated;
};

// Consecutive gated layers keep the shape (stride 1, equal widths), so a run
// of them is one stack: the previous block's epilogue computes the next
// block's mask, and only the run's first block runs a mask launch of its own.
// Returns the run's length (at most kMaxRun) and copies its blocks.
constexpr int32_t kMaxRun = 64;
int32_t gated_run(const dynconv_layer *layers, int32_t i, int32_t n, dynconv_block *blks) {
    int32_t m = 0;
    while (i + m < n && m < kMaxRun && layers[i + m].kind == DYNCONV_LAYER_BLOCK && layers[i + m].gated &&
           layers[i + m].stride == 1 && layers[i + m].blk.c_in == layers[i].blk.c_in &&
           layers[i + m].blk.c_out == layers[i].blk.c_in) {
        blks[m] = layers[i + m].blk;
        ++m;
    }
    return m;
}

dynconv_status net_plan(dynconv_shape in, const dynconv_layer *layers, int32_t n, dynconv_dtype dt,
                        int32_t flags, bool need_mask, NetLayout *NL, dynconv_shape *out_shape,
                        size_t *mask_total) {
    const size_t sz = dtype_size(dt);
    size_t act = 0, h1 = 0, h2 = 0, inner = 0, mtot = 0;
    int ngated = 0;
    dynconv_shape cur = in;
    for (int32_t i = 0; i < n; ++i) {
        LayerShapes ls;
        if (dynconv_status st = layer_shape(layers[i], cur, ls, need_mask)) return st;
        if (dynconv_status st = check_shape(ls.out, true)) return st;
        const size_t npos_in = static_cast<size_t>(positions(ls.in));
        const size_t npos_out = static_cast<size_t>(positions(ls.out));
        act = std::max(act, npos_out * ls.out.c * sz);
        if (layers[i].kind == DYNCONV_LAYER_BLOCK && layers[i].gated) {
            dynconv_block blks[kMaxRun];
            const int32_t m = gated_run(layers, i, n, blks);
            for (int32_t j = 1; j < m; ++j) {  // the run's later layers: checked like any other
                LayerShapes lj;
                if (dynconv_status st = layer_shape(layers[i + j], ls.out, lj, need_mask)) return st;
            }
            ngated += m;
            mtot += static_cast<size_t>(m) * npos_in;
            inner = std::max(inner, stack_layout(ls.in, blks, m, dt, flags).total);
            i += m - 1;
        } else if (layers[i].kind == DYNCONV_LAYER_BLOCK) {
            if (layers[i].blk.w_expand) h1 = std::max(h1, npos_in * ls.hidden * sz);
            h2 = std::max(h2, npos_out * ls.hidden * sz);
        }
        cur = ls.out;
    }
    if (out_shape) *out_shape = cur;
    if (mask_total) *mask_total = mtot;
    if (NL) {
        size_t off = 0;
        NL->act_bytes = act;
        NL->act0 = off; off += align_up(act);
        NL->act1 = off; off += align_up(act);
        NL->h1 = off;   off += align_up(h1);
        NL->h2 = off;   off += align_up(h2);
        NL->masks = off; off += align_up(mtot);
        NL->counts = off; off += align_up(8 * static_cast<size_t>(ngated));
        NL->inner = off; off += inner;
        NL->inner_bytes = inner;
        NL->total = off;
        NL->ngated = ngated;
    }
    return DYNCONV_OK;
}

int elem_grid(int64_t lanes) {
    int64_t g = (lanes + kBlock - 1) / kBlock;
    if (g > 16384) g = 16384;
    if (g < 1) g = 1;
    return static_cast<int>(g);
}

// Workgroups of a kernel that the whole device holds at once (occupancy x
// compute units); 0 when the runtime cannot say.
template <typename K>
int64_t resident_groups(K kern, size_t lds) {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kBlock, lds) != hipSuccess)
        return 0;
    return static_cast<int64_t>(cus) * per_cu;
}

template <typename T, int OT, int KB>
void launch_conv1x1_k(const void *x, int64_t P, int C, const void *w, const float *b, int O, int act,
                      const void *res, void *y, hipStream_t st, Marks &mk) {
    const int nor = ((O + 15) / 16 + OT - 1) / OT;
    const int64_t ptiles = (P + kPwPos - 1) / kPwPos;
    int64_t slots = (ptiles + 7) / 8;  // position-tile slots per XCD
    // one contraction chunk: as many workgroups as the device holds at once
    // (queried once), each staging the weights once and walking several
    // tiles; else one tile per workgroup
    const bool one_chunk = C <= KB * 32;
    static std::atomic<int64_t> resident{0};
    if (one_chunk && resident.load() == 0)
        resident.store(resident_groups(k_conv1x1<T, OT, KB>, pw_lds_bytes<T, OT, KB>()));
    const int64_t full = resident.load() > 0 ? resident.load() : 1024;
    const int64_t cap = one_chunk ? (full / 8 + nor - 1) / nor : 2048 / nor + 1;
    if (slots > cap) slots = cap;
    if (slots < 1) slots = 1;
    launch(mk, k_conv1x1<T, OT, KB>, dim3(static_cast<unsigned>(slots * 8 * nor)), dim3(kBlock),
           pw_lds_bytes<T, OT, KB>(), st, static_cast<const T *>(x), P, C, static_cast<const T *>(w), b, O, act,
           static_cast<const T *>(res), static_cast<T *>(y), nor);
}

// Output tiles per workgroup (2, 4, 6, 8 or 12) and contraction steps per
// chunk (1, 2, 4 or 8): one output range when the outputs fit 12 tiles;
// fewer tiles per range while position tiles x ranges stay under 1024 work
// items; the largest chunk the contraction needs whose staged weights fit
// 64 KB of LDS.
template <typename T, int OT>
void launch_conv1x1_ot(const void *x, int64_t P, int C, const void *w, const float *b, int O, int act,
                       const void *res, void *y, hipStream_t st, Marks &mk) {
    constexpr bool kFits8 = pw_lds_bytes<T, OT, 8>() <= kMaxDynLds;
    const int ks = (C + 31) / 32;
    int kb = ks <= 1 ? 1 : ks <= 2 ? 2 : ks <= 4 ? 4 : 8;
    if (kb == 8 && !kFits8) kb = 4;
    while (kb > 1 && static_cast<size_t>(OT) * 16 * (kb * 32 + 8) * sizeof(T) > kMaxDynLds) kb /= 2;
    if (kb == 1) launch_conv1x1_k<T, OT, 1>(x, P, C, w, b, O, act, res, y, st, mk);
    else if (kb == 2) launch_conv1x1_k<T, OT, 2>(x, P, C, w, b, O, act, res, y, st, mk);
    else if (kb == 4) launch_conv1x1_k<T, OT, 4>(x, P, C, w, b, O, act, res, y, st, mk);
    else if constexpr (kFits8) launch_conv1x1_k<T, OT, 8>(x, P, C, w, b, O, act, res, y, st, mk);
}

template <typename T>
void launch_conv1x1(const void *x, int64_t P, int C, const void *w, const float *b, int O, int act,
                    const void *res, void *y, hipStream_t st, Marks &mk) {
    static const int kOt[] = {12, 8, 6, 4, 2};
    const int nmt = (O + 15) / 16;
    const int64_t ptiles = (P + kPwPos - 1) / kPwPos;
    int i = nmt <= 2 ? 4 : nmt <= 4 ? 3 : nmt <= 6 ? 2 : nmt <= 8 ? 1 : 0;
    while (i < 4 && ptiles * ((nmt + kOt[i] - 1) / kOt[i]) < 1024) ++i;
    switch (kOt[i]) {
    case 12: launch_conv1x1_ot<T, 12>(x, P, C, w, b, O, act, res, y, st, mk); break;
    case 8: launch_conv1x1_ot<T, 8>(x, P, C, w, b, O, act, res, y, st, mk); break;
    case 6: launch_conv1x1_ot<T, 6>(x, P, C, w, b, O, act, res, y, st, mk); break;
    case 4: launch_conv1x1_ot<T, 4>(x, P, C, w, b, O, act, res, y, st, mk); break;
    default: launch_conv1x1_ot<T, 2>(x, P, C, w, b, O, act, res, y, st, mk); break;
    }
}

// Output rows per depthwise task: 4 for 16-bit storage, 2 for fp32.
template <typename T, int S>
void launch_dwconv_s(const void *x, dynconv_shape in, dynconv_shape out, int C, const void *w, const float *b,
                     int act, void *y, hipStream_t st, Marks &mk) {
    constexpr int R = sizeof(T) == 4 ? 2 : 4;
    const size_t lds = static_cast<size_t>(9) * C * sizeof(T);
    const int64_t chunks = (static_cast<int64_t>(out.w) * (C / 8) + kBlock - 1) / kBlock;
    int64_t items = static_cast<int64_t>(out.n) * ((out.h + R - 1) / R) * chunks;
    if (items > 4096) items = 4096;
    if (items < 1) items = 1;
    launch(mk, k_dwconv3x3<T, S, R>, dim3(static_cast<unsigned>(items)), dim3(kBlock), lds, st,
           static_cast<const T *>(x), in.n, in.h, in.w, C, static_cast<const T *>(w), b, act, static_cast<T *>(y),
           out.h, out.w);
}

template <typename T>
void launch_dwconv(const void *x, dynconv_shape in, dynconv_shape out, int C, int stride, const void *w,
                   const float *b, int act, void *y, hipStream_t st, Marks &mk) {
    if (stride == 1) launch_dwconv_s<T, 1>(x, in, out, C, w, b, act, y, st, mk);
    else launch_dwconv_s<T, 2>(x, in, out, C, w, b, act, y, st, mk);
}

template <typename T, int KS, int OT>
void launch_conv3x3_mfma(const void *x, dynconv_shape in, dynconv_shape out, const dynconv_layer &L, void *y,
                         hipStream_t st, Marks &mk) {
    const size_t lds = static_cast<size_t>(L.c_out) * (KS * 32 + 8) * sizeof(T) + 4 * 32 * KS;
    int64_t grid = (positions(out) + 63) / 64;
    if (grid > 8192) grid = 8192;
    if (grid < 1) grid = 1;
    launch(mk, k_conv3x3_mfma<T, KS, OT>, dim3(static_cast<unsigned>(grid)), dim3(kBlock), lds, st,
           static_cast<const T *>(x), in.n, in.h, in.w, L.c_in, L.stride, static_cast<const T *>(L.w), L.b,
           L.c_out, L.act, static_cast<T *>(y), out.h, out.w);
}

// 16-bit storage: the matrix-core form when its weights fit 64 KB of LDS;
// fp32 (and wider layers): one lane per position on the VALU.
template <typename T>
void launch_conv3x3(const void *x, dynconv_shape in, dynconv_shape out, const dynconv_layer &L, void *y,
                    hipStream_t st, Marks &mk) {
    const int ks = (9 * L.c_in + 31) / 32;
    if constexpr (sizeof(T) == 2) {
        const size_t lds = static_cast<size_t>(L.c_out) * (ks * 32 + 8) * sizeof(T) + 4 * 32 * ks;
        if (lds <= kMaxDynLds) {
            const bool wide = L.c_out > 32;
#define DC_C3(KS)                                                                         \
    (wide ? launch_conv3x3_mfma<T, KS, 4>(x, in, out, L, y, st, mk)                      \
          : launch_conv3x3_mfma<T, KS, 2>(x, in, out, L, y, st, mk))
            switch (ks) {
            case 1: DC_C3(1); return;
            case 2: DC_C3(2); return;
            case 3: DC_C3(3); return;
            case 4: DC_C3(4); return;
            case 5: DC_C3(5); return;
            default: break;
            }
#undef DC_C3
        }
    }
    const size_t lds = 4 * (9 * L.c_in * L.c_out + L.c_out);
    launch(mk, k_conv3x3<T>, dim3(elem_grid(positions(out))), dim3(kBlock), lds, st,
           static_cast<const T *>(x), in.n, in.h, in.w, L.c_in, L.stride, static_cast<const T *>(L.w), L.b,
           L.c_out, L.act, static_cast<T *>(y), out.h, out.w);
}

// Expansion + depthwise in one launch (ungated blocks): 16-bit storage, at
// most 64 input channels, LDS within 64 KB, and at least kEdMinItems 8x8
// output tiles (below that too few workgroups share the work; MobileNetV2
// at batch 64: 112x112x16 -> 96 and 56x56x24 -> 144 qualify, 62 against 100
// us and 38 against 41 us with the projection).
constexpr int64_t kEdMinItems = 1024;

int64_t ed_items(dynconv_shape out) {
    return static_cast<int64_t>(out.n) * ((out.h + kEdTile - 1) / kEdTile) * ((out.w + kEdTile - 1) / kEdTile);
}

bool use_expand_dw(dynconv_dtype dt, int C, int E, int stride, dynconv_shape out) {
    if (dt == DYNCONV_F32 || C > 64 || ed_items(out) < kEdMinItems) return false;
    const size_t lds = stride == 1 ? ed_lds_bytes<half_t, 1>(C, E) : ed_lds_bytes<half_t, 2>(C, E);
    return lds <= kMaxDynLds;
}

// Persistent workgroups: as many as the device holds at once.
template <typename T, int S, int KS>
void launch_expand_dw_k(const void *x, dynconv_shape in, dynconv_shape out, const dynconv_block &b, int E,
                        void *h2, hipStream_t st, Marks &mk) {
    const size_t lds = ed_lds_bytes<T, S>(b.c_in, E);
    int64_t grid = ed_items(out);
    const int64_t full = resident_groups(k_expand_dw<T, S, KS>, lds);
    if (full > 0 && grid > full) grid = full;
    launch(mk, k_expand_dw<T, S, KS>, dim3(static_cast<unsigned>(grid)), dim3(kBlock), lds,
           st, static_cast<const T *>(x), in.n, in.h, in.w, b.c_in, static_cast<const T *>(b.w_expand), b.b_expand,
           b.act_expand, E, static_cast<const T *>(b.w_dw), b.b_dw, b.act_dw, static_cast<T *>(h2), out.h, out.w);
}

template <typename T>
void launch_expand_dw(const void *x, dynconv_shape in, dynconv_shape out, const dynconv_block &b, int E, int stride,
                      void *h2, hipStream_t st, Marks &mk) {
    if constexpr (sizeof(T) == 2) {
        const bool k1 = b.c_in <= 32;
        if (stride == 1) {
            if (k1) launch_expand_dw_k<T, 1, 1>(x, in, out, b, E, h2, st, mk);
            else launch_expand_dw_k<T, 1, 2>(x, in, out, b, E, h2, st, mk);
        } else {
            if (k1) launch_expand_dw_k<T, 2, 1>(x, in, out, b, E, h2, st, mk);
            else launch_expand_dw_k<T, 2, 2>(x, in, out, b, E, h2, st, mk);
        }
    }
}

#define DC_TYPED(dt, call)                                  \
    do {                                                    \
        if ((dt) == DYNCONV_F32) { typedef float T; call; }  \
        else if ((dt) == DYNCONV_F16) { typedef half_t T; call; } \
        else { typedef bf16_t T; call; }                    \
    } while (0)

void net_walk(const void *x, void *y, dynconv_shape in, dynconv_dtype dt, const dynconv_layer *layers,
              int32_t n, int32_t flags, uint8_t *masks, int32_t *counts, char *base, const NetLayout &NL,
              hipStream_t st, Marks &mk, Plan &plan) {
    void *bufs[2] = {at(base, NL.act0), at(base, NL.act1)};
    void *h1 = at(base, NL.h1), *h2 = at(base, NL.h2);
    char *inner = at(base, NL.inner);
    dynconv_shape cur = in;
    const void *src = x;
    size_t moff = 0;
    int gi = 0;
    for (int32_t i = 0; i < n; ++i) {
        const dynconv_layer &L = layers[i];
        LayerShapes ls;
        layer_shape(L, cur, ls, false);
        void *dst = (i == n - 1) ? y : bufs[i % 2];
        if (L.kind == DYNCONV_LAYER_CONV3X3) {
            if (plan.note("k_conv3x3")) DC_TYPED(dt, launch_conv3x3<T>(src, ls.in, ls.out, L, dst, st, mk));
        } else if (L.kind == DYNCONV_LAYER_CONV1X1) {
            if (plan.note("k_conv1x1"))
                DC_TYPED(dt, launch_conv1x1<T>(src, positions(ls.in), L.c_in, L.w, L.b, L.c_out, L.act, nullptr,
                                               dst, st, mk));
        } else if (L.gated) {
            dynconv_block blks[kMaxRun];
            const int32_t m = gated_run(layers, i, n, blks);
            i += m - 1;  // the run's last layer
            dst = (i == n - 1) ? y : bufs[i % 2];
            StackLayout SL = stack_layout(ls.in, blks, m, dt, flags);
            uint8_t *mk_l = masks ? masks + moff : nullptr;
            int32_t *ct_l = counts ? counts + 2 * gi : nullptr;
            stack_walk(src, dst, ls.in, dt, blks, m, flags, mk_l, ct_l, inner, SL, st, mk, plan, dst == src);
            moff += static_cast<size_t>(m) * positions(ls.in);
            gi += m;
        } else {
            const dynconv_block &b = L.blk;
            const void *hin = src;
            if (b.w_expand && use_expand_dw(dt, b.c_in, ls.hidden, L.stride, ls.out)) {
                if (plan.note("k_expand_dw"))
                    DC_TYPED(dt, launch_expand_dw<T>(src, ls.in, ls.out, b, ls.hidden, L.stride, h2, st, mk));
                const bool resid = L.stride == 1 && b.c_in == b.c_out;
                if (plan.note("k_conv1x1"))
                    DC_TYPED(dt, launch_conv1x1<T>(h2, positions(ls.out), ls.hidden, b.w_project, b.b_project,
                                                   b.c_out, b.act_project, resid ? src : nullptr, dst, st, mk));
                src = dst;
                cur = ls.out;
                continue;
            }
            if (b.w_expand) {
                if (plan.note("k_conv1x1"))
                    DC_TYPED(dt, launch_conv1x1<T>(src, positions(ls.in), b.c_in, b.w_expand, b.b_expand,
                                                   ls.hidden, b.act_expand, nullptr, h1, st, mk));
                hin = h1;
            }
            dynconv_shape hs = ls.in;
            hs.c = ls.hidden;
            if (plan.note("k_dwconv3x3"))
                DC_TYPED(dt, launch_dwconv<T>(hin, hs, ls.out, ls.hidden, L.stride, b.w_dw, b.b_dw, b.act_dw, h2,
                                              st, mk));
            const bool resid = L.stride == 1 && b.c_in == b.c_out;
            if (plan.note("k_conv1x1"))
                DC_TYPED(dt, launch_conv1x1<T>(h2, positions(ls.out), ls.hidden, b.w_project, b.b_project,
                                               b.c_out, b.act_project, resid ? src : nullptr, dst, st, mk));
        }
        src = dst;
        cur = ls.out;
    }
}

// ------------------------------------------------------------ static scratch
// Device memory of the stack call that allocates nothing: one array per
// device, held until the process ends.  In host code `scratch` names a
// host-side stand-in, never a device address: kernels and copies take the
// address that hipGetSymbolAddress returns for the current device.
constexpr size_t kStaticScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) char scratch[kStaticScratchBytes];
std::atomic<char *> g_scratch_ptr[kMaxDevices];

// The current device's copy of `scratch` (looked up once per device).
dynconv_status static_scratch(char **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return DYNCONV_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return DYNCONV_ERR_UNSUPPORTED;
    char *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        void *q = nullptr;
        if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return DYNCONV_ERR_HIP;
        p = static_cast<char *>(q);
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return DYNCONV_OK;
}

}  // namespace

// ================================================================ C ABI
extern "C" {

const char *dynconv_status_str(int32_t status) {
    switch (status) {
    case DYNCONV_OK: return "ok";
    case DYNCONV_ERR_NULL: return "required pointer is NULL";
    case DYNCONV_ERR_SHAPE: return "invalid shape or overlapping buffers";
    case DYNCONV_ERR_DTYPE: return "unknown dtype";
    case DYNCONV_ERR_UNSUPPORTED: return "shape or channel count not supported by the kernels";
    case DYNCONV_ERR_CAPACITY: return "index buffers smaller than N*H*W";
    case DYNCONV_ERR_ALIGN: return "data pointer not 16-byte aligned";
    case DYNCONV_ERR_WORKSPACE: return "workspace missing or too small";
    case DYNCONV_ERR_HIP: return "HIP launch failed";
    case DYNCONV_ERR_ARG: return "argument out of range";
    }
    return "unknown status";
}

const char *dynconv_version(void) { return "dynconv-mi355x 0.1 (gfx950)"; }

static dynconv_status mask_common(const void *x, dynconv_shape s, dynconv_dtype dt, const float *w_mask,
                                  float b_mask, uint8_t *mask, float *logits, int mode, void *stream) {
    if (!x || !w_mask || !mask) return DYNCONV_ERR_NULL;
    if (!dtype_ok(dt)) return DYNCONV_ERR_DTYPE;
    if (dynconv_status st = check_shape(s, true)) return st;
    if (dynconv_status st = check_channels(s.c)) return st;
    if (!aligned16(x)) return DYNCONV_ERR_ALIGN;
    (void)hipGetLastError();
    Marks mk;
    dispatch_mask(dt, x, s, w_mask, b_mask, mask, logits, mode, static_cast<hipStream_t>(stream), mk);
    return launch_status();
}

dynconv_status dynconv_mask(const void *x, dynconv_shape s, dynconv_dtype dt, const float *w_mask,
                            float b_mask, uint8_t *mask, float *logits, void *stream) {
    return mask_common(x, s, dt, w_mask, b_mask, mask, logits, 0, stream);
}

dynconv_status dynconv_mask_gsoftmax(const void *x, dynconv_shape s, dynconv_dtype dt,
                                     const float *w_mask, float b_mask, uint8_t *mask, float *logits,
                                     void *stream) {
    return mask_common(x, s, dt, w_mask, b_mask, mask, logits, 1, stream);
}

size_t dynconv_indices_workspace_bytes(dynconv_shape s) {
    if (check_shape(s, false) != DYNCONV_OK) return 0;
    return index_scratch_bytes(s);
}

dynconv_status dynconv_build_indices(const uint8_t *mask, dynconv_shape s, int32_t dilate,
                                     const dynconv_indices *idx, void *ws, size_t ws_bytes,
                                     void *stream) {
    if (!mask || !idx) return DYNCONV_ERR_NULL;
    if (!idx->active || !idx->dilated || !idx->nbr || !idx->counts) return DYNCONV_ERR_NULL;
    if (dynconv_status st = check_shape(s, false)) return st;
    if (dilate < 0 || dilate > kMaxDilate) return DYNCONV_ERR_ARG;
    if (idx->capacity < positions(s)) return DYNCONV_ERR_CAPACITY;
    if (!ws || ws_bytes < index_scratch_bytes(s)) return DYNCONV_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(ws) & 7u) != 0) return DYNCONV_ERR_ALIGN;
    (void)hipGetLastError();
    Marks mk;
    launch_indices(mask, s, dilate, idx, ws, static_cast<hipStream_t>(stream), mk);
    return launch_status();
}

size_t dynconv_block_workspace_bytes(dynconv_shape s, const dynconv_block *blk, dynconv_dtype dt) {
    if (!blk || !dtype_ok(dt) || check_shape(s, true) != DYNCONV_OK || blk->c_hidden <= 0) return 0;
    return hidden_bytes(s, blk->c_hidden, dt);
}

dynconv_status dynconv_block_forward(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                     const dynconv_block *blk, const dynconv_indices *idx, void *ws,
                                     size_t ws_bytes, void *stream) {
    if (!x || !y) return DYNCONV_ERR_NULL;
    if (!dtype_ok(dt)) return DYNCONV_ERR_DTYPE;
    if (dynconv_status st = check_shape(s, true)) return st;
    if (dynconv_status st = check_block(blk, s, false)) return st;
    if (!aligned16(x) || !aligned16(y)) return DYNCONV_ERR_ALIGN;
    size_t bytes = static_cast<size_t>(positions(s)) * s.c * dtype_size(dt);
    if (x != y && ranges_overlap(x, bytes, y, bytes)) return DYNCONV_ERR_SHAPE;
    if (idx) {
        if (!idx->active || !idx->dilated || !idx->nbr || !idx->counts) return DYNCONV_ERR_NULL;
        if (idx->capacity < positions(s)) return DYNCONV_ERR_CAPACITY;
    }
    if (!ws || ws_bytes < hidden_bytes(s, blk->c_hidden, dt)) return DYNCONV_ERR_WORKSPACE;
    if (!aligned16(ws)) return DYNCONV_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    Marks mk;
    if (x != y) launch_copy(x, y, bytes, st, mk);
    dispatch_block(dt, x, y, s, blk, idx, ws, st, mk);
    return launch_status();
}

size_t dynconv_stack_workspace_bytes(dynconv_shape s, const dynconv_block *blks, int32_t n_blocks,
                                     dynconv_dtype dt, int32_t flags) {
    if (!blks || n_blocks < 1 || n_blocks > kMaxBlocks || !dtype_ok(dt) ||
        check_shape(s, true) != DYNCONV_OK)
        return 0;
    return stack_layout(s, blks, n_blocks, dt, flags).total;
}

static dynconv_status stack_common(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                   const dynconv_block *blks, int32_t n_blocks, int32_t flags,
                                   uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                   void *stream, void *const *events, int32_t n_events,
                                   bool profiled) {
    if (dynconv_status st = stack_checked(x, y, s, dt, blks, n_blocks, flags)) return st;
    StackLayout L = stack_layout(s, blks, n_blocks, dt, flags);
    if (!ws || ws_bytes < L.total) return DYNCONV_ERR_WORKSPACE;
    if (!aligned16(ws)) return DYNCONV_ERR_ALIGN;
    const bool in_place = x == y;
    Marks mk;
    if (profiled) {
        Plan count{false, nullptr, 0};
        StackLayout L0 = L;
        Marks none;
        stack_walk(x, y, s, dt, blks, n_blocks, flags, masks, counts, nullptr, L0, nullptr, none,
                   count, in_place);
        if (!events) return DYNCONV_ERR_NULL;
        if (n_events < 2 * count.count) return DYNCONV_ERR_ARG;
        for (int32_t i = 0; i < 2 * count.count; ++i)
            if (!events[i]) return DYNCONV_ERR_NULL;
        mk.ev = reinterpret_cast<hipEvent_t const *>(events);
        mk.n = 2 * count.count;
    }
    (void)hipGetLastError();
    Plan run{true, nullptr, 0};
    stack_walk(x, y, s, dt, blks, n_blocks, flags, masks, counts, static_cast<char *>(ws), L,
               static_cast<hipStream_t>(stream), mk, run, in_place);
    return launch_status();
}

dynconv_status dynconv_stack_forward(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                     const dynconv_block *blks, int32_t n_blocks, int32_t flags,
                                     uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                     void *stream) {
    return stack_common(x, y, s, dt, blks, n_blocks, flags, masks, counts, ws, ws_bytes, stream,
                        nullptr, 0, false);
}

int32_t dynconv_stack_launch_names(dynconv_shape s, const dynconv_block *blks, int32_t n_blocks,
                                   dynconv_dtype dt, int32_t flags, int32_t in_place,
                                   const char **names, int32_t cap) {
    if (!blks || n_blocks < 1 || n_blocks > kMaxBlocks || !dtype_ok(dt) ||
        check_shape(s, true) != DYNCONV_OK || (flags & ~kStackFlags))
        return -1;
    StackLayout L = stack_layout(s, blks, n_blocks, dt, flags);
    Plan plan{false, names, names ? cap : 0};
    Marks none;
    stack_walk(nullptr, nullptr, s, dt, blks, n_blocks, flags, nullptr, nullptr, nullptr, L,
               nullptr, none, plan, in_place != 0);
    return plan.count;
}

dynconv_status dynconv_stack_forward_profiled(const void *x, void *y, dynconv_shape s,
                                              dynconv_dtype dt, const dynconv_block *blks,
                                              int32_t n_blocks, int32_t flags, uint8_t *masks,
                                              int32_t *counts, void *ws, size_t ws_bytes,
                                              void *stream, void *const *events, int32_t n_events) {
    return stack_common(x, y, s, dt, blks, n_blocks, flags, masks, counts, ws, ws_bytes, stream,
                        events, n_events, true);
}

size_t dynconv_stack_noalloc_max_workspace_bytes(void) { return kStaticScratchBytes; }

dynconv_status dynconv_stack_forward_noalloc(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                             const dynconv_block *blks, int32_t n_blocks, int32_t flags,
                                             uint8_t *masks, int32_t *counts, void *stream) {
    if (dynconv_status st = stack_checked(x, y, s, dt, blks, n_blocks, flags)) return st;
    if (stack_layout(s, blks, n_blocks, dt, flags).total > kStaticScratchBytes) return DYNCONV_ERR_WORKSPACE;
    char *ws = nullptr;
    if (dynconv_status st = static_scratch(&ws)) return st;
    return stack_common(x, y, s, dt, blks, n_blocks, flags, masks, counts, ws, kStaticScratchBytes, stream,
                        nullptr, 0, false);
}

size_t dynconv_shuffle_stack_workspace_bytes(dynconv_shape s, const dynconv_block *branches,
                                             int32_t n_units, dynconv_dtype dt, int32_t flags) {
    if (!branches || n_units < 1 || n_units > kMaxBlocks || !dtype_ok(dt) ||
        check_shape(s, true) != DYNCONV_OK || s.c % 2 != 0 || branches[0].c_in <= 0)
        return 0;
    return shuffle_layout(s, branches, n_units, dt, flags).total;
}

static dynconv_status shuffle_common(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                     const dynconv_block *br, int32_t n_units, int32_t flags,
                                     uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                     void *stream, void *const *events, int32_t n_events,
                                     bool profiled) {
    if (dynconv_status st = shuffle_checked(x, y, s, dt, br, n_units, flags)) return st;
    ShuffleLayout L = shuffle_layout(s, br, n_units, dt, flags);
    if (!ws || ws_bytes < L.total) return DYNCONV_ERR_WORKSPACE;
    if (!aligned16(ws)) return DYNCONV_ERR_ALIGN;
    Marks mk;
    if (profiled) {
        Plan count{false, nullptr, 0};
        Marks none;
        shuffle_walk(x, y, s, dt, br, n_units, flags, masks, counts, nullptr, L, nullptr, none, count);
        if (!events) return DYNCONV_ERR_NULL;
        if (n_events < 2 * count.count) return DYNCONV_ERR_ARG;
        for (int32_t i = 0; i < 2 * count.count; ++i)
            if (!events[i]) return DYNCONV_ERR_NULL;
        mk.ev = reinterpret_cast<hipEvent_t const *>(events);
        mk.n = 2 * count.count;
    }
    (void)hipGetLastError();
    Plan run{true, nullptr, 0};
    shuffle_walk(x, y, s, dt, br, n_units, flags, masks, counts, static_cast<char *>(ws), L,
                 static_cast<hipStream_t>(stream), mk, run);
    return launch_status();
}

dynconv_status dynconv_shuffle_stack_forward(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                             const dynconv_block *branches, int32_t n_units,
                                             int32_t flags, uint8_t *masks, int32_t *counts, void *ws,
                                             size_t ws_bytes, void *stream) {
    return shuffle_common(x, y, s, dt, branches, n_units, flags, masks, counts, ws, ws_bytes, stream,
                          nullptr, 0, false);
}

int32_t dynconv_shuffle_stack_launch_names(dynconv_shape s, const dynconv_block *branches,
                                           int32_t n_units, dynconv_dtype dt, int32_t flags,
                                           const char **names, int32_t cap) {
    if (!branches || n_units < 1 || n_units > kMaxBlocks || !dtype_ok(dt) ||
        check_shape(s, true) != DYNCONV_OK || s.c % 2 != 0 || branches[0].c_in <= 0 ||
        (flags & ~kStackFlags))
        return -1;
    ShuffleLayout L = shuffle_layout(s, branches, n_units, dt, flags);
    Plan plan{false, names, names ? cap : 0};
    Marks none;
    shuffle_walk(nullptr, nullptr, s, dt, branches, n_units, flags, nullptr, nullptr, nullptr, L, nullptr,
                 none, plan);
    return plan.count;
}

dynconv_status dynconv_shuffle_stack_forward_profiled(const void *x, void *y, dynconv_shape s,
                                                      dynconv_dtype dt, const dynconv_block *branches,
                                                      int32_t n_units, int32_t flags, uint8_t *masks,
                                                      int32_t *counts, void *ws, size_t ws_bytes,
                                                      void *stream, void *const *events,
                                                      int32_t n_events) {
    return shuffle_common(x, y, s, dt, branches, n_units, flags, masks, counts, ws, ws_bytes, stream,
                          events, n_events, true);
}

dynconv_status dynconv_network_output_shape(dynconv_shape in, const dynconv_layer *layers, int32_t n_layers,
                                            dynconv_shape *out) {
    if (!layers || !out) return DYNCONV_ERR_NULL;
    if (n_layers < 1 || n_layers > kMaxLayers) return DYNCONV_ERR_ARG;
    if (dynconv_status st = check_shape(in, true)) return st;
    return net_plan(in, layers, n_layers, DYNCONV_F16, 0, false, nullptr, out, nullptr);
}

size_t dynconv_network_workspace_bytes(dynconv_shape in, const dynconv_layer *layers, int32_t n_layers,
                                       dynconv_dtype dt, int32_t flags) {
    if (!layers || n_layers < 1 || n_layers > kMaxLayers || !dtype_ok(dt) || check_shape(in, true) != DYNCONV_OK ||
        (flags & ~kStackFlags))
        return 0;
    NetLayout NL;
    if (net_plan(in, layers, n_layers, dt, flags, false, &NL, nullptr, nullptr) != DYNCONV_OK) return 0;
    return NL.total;
}

static dynconv_status net_common(const void *x, void *y, dynconv_shape in, dynconv_dtype dt,
                                 const dynconv_layer *layers, int32_t n, int32_t flags, uint8_t *masks,
                                 int32_t *counts, void *ws, size_t ws_bytes, void *stream,
                                 void *const *events, int32_t n_events, bool profiled) {
    if (!x || !y || !layers) return DYNCONV_ERR_NULL;
    if (!dtype_ok(dt)) return DYNCONV_ERR_DTYPE;
    if (n < 1 || n > kMaxLayers) return DYNCONV_ERR_ARG;
    if (flags & ~kStackFlags) return DYNCONV_ERR_ARG;
    if (dynconv_status st = check_shape(in, true)) return st;
    NetLayout NL;
    dynconv_shape out;
    if (dynconv_status st = net_plan(in, layers, n, dt, flags, !(flags & kStackDense), &NL, &out, nullptr))
        return st;
    if (!aligned16(x) || !aligned16(y)) return DYNCONV_ERR_ALIGN;
    const size_t in_bytes = static_cast<size_t>(positions(in)) * in.c * dtype_size(dt);
    const size_t out_bytes = static_cast<size_t>(positions(out)) * out.c * dtype_size(dt);
    if (ranges_overlap(x, in_bytes, y, out_bytes)) return DYNCONV_ERR_SHAPE;
    if (!ws || ws_bytes < NL.total) return DYNCONV_ERR_WORKSPACE;
    if (!aligned16(ws)) return DYNCONV_ERR_ALIGN;
    Marks mk;
    if (profiled) {
        Plan count{false, nullptr, 0};
        count.list_counts = counts != nullptr;
        Marks none;
        net_walk(x, y, in, dt, layers, n, flags, masks, counts, nullptr, NL, nullptr, none, count);
        if (!events) return DYNCONV_ERR_NULL;
        if (n_events < 2 * count.count) return DYNCONV_ERR_ARG;
        for (int32_t i = 0; i < 2 * count.count; ++i)
            if (!events[i]) return DYNCONV_ERR_NULL;
        mk.ev = reinterpret_cast<hipEvent_t const *>(events);
        mk.n = 2 * count.count;
    }
    (void)hipGetLastError();
    Plan run{true, nullptr, 0};
    net_walk(x, y, in, dt, layers, n, flags, masks, counts, static_cast<char *>(ws), NL,
             static_cast<hipStream_t>(stream), mk, run);
    return launch_status();
}

dynconv_status dynconv_network_forward(const void *x, void *y, dynconv_shape in, dynconv_dtype dt,
                                       const dynconv_layer *layers, int32_t n_layers, int32_t flags,
                                       uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                       void *stream) {
    return net_common(x, y, in, dt, layers, n_layers, flags, masks, counts, ws, ws_bytes, stream, nullptr, 0,
                      false);
}

int32_t dynconv_network_launch_names(dynconv_shape in, const dynconv_layer *layers, int32_t n_layers,
                                     dynconv_dtype dt, int32_t flags, int32_t with_counts, const char **names,
                                     int32_t cap) {
    if (!layers || n_layers < 1 || n_layers > kMaxLayers || !dtype_ok(dt) || check_shape(in, true) != DYNCONV_OK ||
        (flags & ~kStackFlags))
        return -1;
    NetLayout NL;
    if (net_plan(in, layers, n_layers, dt, flags, false, &NL, nullptr, nullptr) != DYNCONV_OK) return -1;
    Plan plan{false, names, names ? cap : 0};
    plan.list_counts = with_counts != 0;
    Marks none;
    net_walk(nullptr, nullptr, in, dt, layers, n_layers, flags, nullptr, nullptr, nullptr, NL, nullptr, none,
             plan);
    return plan.count;
}

dynconv_status dynconv_network_forward_profiled(const void *x, void *y, dynconv_shape in, dynconv_dtype dt,
                                                const dynconv_layer *layers, int32_t n_layers, int32_t flags,
                                                uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                                void *stream, void *const *events, int32_t n_events) {
    return net_common(x, y, in, dt, layers, n_layers, flags, masks, counts, ws, ws_bytes, stream, events,
                      n_events, true);
}

}  // extern "C"
