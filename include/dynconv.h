/*
 * dynconv.h -- C ABI of the MI355X (gfx950) library for spatially gated
 * MobileNetV2 inverted-residual blocks: the inference path of Verelst &
 * Tuytelaars, "Dynamic Convolutions: Exploiting Spatial Sparsity for Faster
 * Inference" (CVPR 2020), Sec. 3.1.1 (block and mask unit), Sec. 3.1.2 (hard
 * decision) and Sec. 3.2 (gather / modified depthwise / scatter execution).
 *
 * Conventions shared by every call
 * --------------------------------
 * * Feature maps are NHWC, dense, channel fastest: element (n, h, w, c) sits
 *   at ((n*H + h)*W + w)*C + c.  Flat positions are raster ordered,
 *   i = (n*H + h)*W + w, image-major; the paper's "p-th active position of the
 *   flattened mask" uses this order (Sec. 3.2, masked gather).
 * * Pointers marked (device) must be device memory of the current HIP device;
 *   (host) pointers are read during the call only.  The library allocates and
 *   frees nothing: every buffer, including the workspace, belongs to the
 *   caller.  Its only global state is a cache of device occupancy figures
 *   (workgroups the device holds at once, per kernel; written once, read
 *   atomically) and the static scratch array of
 *   dynconv_stack_forward_noalloc, so calls on different streams may run
 *   concurrently as long as their buffers are disjoint (for that call: as
 *   long as they run on different devices).
 * * Every call validates all of its arguments on the host first.  On any
 *   error it returns a nonzero status and enqueues nothing.  Otherwise the
 *   work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *   null stream) and DYNCONV_OK is returned; a failed kernel launch is
 *   reported as DYNCONV_ERR_HIP (the call clears HIP's last-error state
 *   before launching).  Nothing synchronises with the host, nothing is
 *   printed, no exception leaves the library.  No call enqueues a memset or
 *   a host synchronisation, so the calls may be captured into a HIP graph.
 * * Sizes that the mask decides (the active count P and the dilated count
 *   P_d) stay on the device; kernels are sized for the capacity N*H*W and
 *   read the counts there.
 * * Data types: fp32, fp16 and bf16 storage.  Arithmetic is fp32 (fp32
 *   accumulation in the matrix-core products); the expanded and depthwise
 *   intermediates are rounded to the storage type.
 * * Supported channel counts: c_in == c_out (the identity path of Eq. 3),
 *   8 <= c_in <= 256 with c_in % 8 == 0, 16 <= c_hidden <= 1536 with
 *   c_hidden % 16 == 0.  Other valid shapes return DYNCONV_ERR_UNSUPPORTED.
 *   N*H*W must stay below 2^31 / 9.  Data pointers must be 16-byte aligned.
 */
#ifndef DYNCONV_H_
#define DYNCONV_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enumerations are 32-bit integers on both sides of the ABI.  C++ gets a
 * fixed underlying type, so that a caller's out-of-range code (rejected with
 * DYNCONV_ERR_DTYPE) is a defined value there too. */
#ifdef __cplusplus
#define DYNCONV_ENUM(tag) enum tag : int32_t
#else
#define DYNCONV_ENUM(tag) enum tag
#endif

typedef DYNCONV_ENUM(dynconv_dtype_e) {
    DYNCONV_F32 = 0,
    DYNCONV_F16 = 1,
    DYNCONV_BF16 = 2
} dynconv_dtype;

typedef DYNCONV_ENUM(dynconv_status_e) {
    DYNCONV_OK = 0,
    DYNCONV_ERR_NULL = 1,        /* a required pointer is NULL */
    DYNCONV_ERR_SHAPE = 2,       /* non-positive / overflowing sizes, overlapping buffers */
    DYNCONV_ERR_DTYPE = 3,       /* unknown dtype */
    DYNCONV_ERR_UNSUPPORTED = 4, /* well-formed but outside what the kernels implement */
    DYNCONV_ERR_CAPACITY = 5,    /* index buffers hold fewer than N*H*W entries */
    DYNCONV_ERR_ALIGN = 6,       /* a data pointer is not 16-byte aligned */
    DYNCONV_ERR_WORKSPACE = 7,   /* workspace NULL or smaller than required */
    DYNCONV_ERR_HIP = 8,         /* a HIP launch failed */
    DYNCONV_ERR_ARG = 9          /* another argument is out of range (dilation, activation, block count) */
} dynconv_status;

typedef DYNCONV_ENUM(dynconv_act_e) {
    DYNCONV_ACT_NONE = 0,
    DYNCONV_ACT_RELU = 1,
    DYNCONV_ACT_RELU6 = 2
} dynconv_act;

/* Shape of a feature map: n images of h x w positions and c channels. */
typedef struct {
    int32_t n, h, w, c;
} dynconv_shape;

/*
 * One inverted-residual block with batch norm folded into weights and biases
 * (Sec. 3.2: pointwise expansion, depthwise 3x3, linear pointwise
 * projection), plus its 1x1 mask unit (Sec. 3.1.1).  All pointers (device).
 * Weight layouts are PyTorch's convolution layouts, in the storage dtype:
 *   w_expand  [c_hidden][c_in]    (from [E, C, 1, 1])
 *   w_dw      [c_hidden][9]       (from [E, 1, 3, 3]; tap k = 3*(dh+1) + (dw+1))
 *   w_project [c_out][c_hidden]   (from [Co, E, 1, 1])
 * Biases are fp32.  The mask unit is an fp32 weight vector w_mask [c_in] and
 * a scalar b_mask; MobileNetV2 uses act_expand = act_dw = RELU6 and
 * act_project = NONE.
 */
typedef struct {
    int32_t c_in, c_hidden, c_out;
    const void *w_expand;
    const float *b_expand;
    const void *w_dw;
    const float *b_dw;
    const void *w_project;
    const float *b_project;
    int32_t act_expand, act_dw, act_project;
    const float *w_mask;
    float b_mask;
} dynconv_block;

/*
 * Index maps of one hard mask (Sec. 3.2).  All arrays (device), int32, each
 * with room for `capacity` >= N*H*W positions (nbr: 9*capacity entries):
 *   active [P]     ascending flat positions with G = 1
 *   dilated[P_d]   ascending flat positions with G_dilated = 1
 *   nbr    [P][9]  nbr[p*9 + 3*(dh+1) + (dw+1)] = row of `dilated` holding the
 *                  neighbour (h+dh, w+dw) of active[p], or -1 when it lies
 *                  outside the image or outside the dilated mask
 *   counts [2]     P, P_d
 * Entries past the counts are left unspecified.
 */
typedef struct {
    int32_t *active;
    int32_t *dilated;
    int32_t *nbr;
    int32_t *counts;
    int64_t capacity;
} dynconv_indices;

/* Text for a status code, a dynconv_status value passed as an integer so
 * that any code is accepted (static storage, never NULL; codes outside the
 * enumeration give "unknown status"). */
const char *dynconv_status_str(int32_t status);

/* Library identification string (static storage). */
const char *dynconv_version(void);

/*
 * Mask unit and hard decision (Sec. 3.1.1, Eq. 2; Sec. 3.1.2, Eq. 8 with the
 * Gumbel noise fixed to zero at inference):
 *   m[i] = (sum over c ascending of w_mask[c] * x[i, c], as an fp32 fused
 *           multiply-add chain starting from +0) + b_mask     (fp32)
 *   mask[i] = m[i] > 0 ? 1 : 0                                 (ties, NaN -> 0)
 *   x       (device) NHWC, dtype dt, shape s
 *   w_mask  (device) fp32 [s.c]
 *   mask    (device) uint8 [N*H*W], written
 *   logits  (device) fp32 [N*H*W] or NULL, written when non-NULL
 * The fp32 operation order is fixed, so masks are reproducible bit for bit.
 */
dynconv_status dynconv_mask(const void *x, dynconv_shape s, dynconv_dtype dt,
                            const float *w_mask, float b_mask,
                            uint8_t *mask, float *logits, void *stream);

/*
 * The same mask unit with the G-Softmax hard decision at inference
 * (Sec. 3.1.2, the variant of Table 1 that keeps the softmax and the
 * logarithms): with m as above (fp32),
 *   p1 = 1 / (1 + exp(-m)),  p2 = 1 - p1          (Eq. 6, Eq. 7)
 *   y1 = exp(log p1) / (exp(log p1) + exp(log p2))  (Eq. 5, zero noise, tau = 1)
 *   mask[i] = y1 > 1/2 ? 1 : 0
 * in fp32 with the device's expf and logf.  In exact arithmetic y1 = p1 and
 * the decision equals dynconv_mask's; in fp32 the two differ only where the
 * rounding of p1 near 1/2 decides, i.e. for |m| below about 1e-7.
 * Arguments, logits and errors as dynconv_mask.
 */
dynconv_status dynconv_mask_gsoftmax(const void *x, dynconv_shape s, dynconv_dtype dt,
                                     const float *w_mask, float b_mask, uint8_t *mask, float *logits,
                                     void *stream);

/* Workspace bytes that dynconv_build_indices needs for shape s. */
size_t dynconv_indices_workspace_bytes(dynconv_shape s);

/*
 * Mask dilation and index maps, the paper's "bookkeeping" (Sec. 3.2, mask
 * dilation and masked gather; Table 2): the (2*dilate+1)^2 square dilation
 * of the mask within each image, then the raster-ordered lists and the
 * neighbour table described at dynconv_indices.  Output is unique, so it is
 * bit-exact and deterministic.
 *   mask    (device) uint8 [N*H*W] (nonzero = active); s.c is ignored
 *   dilate  0..3; block execution needs 1 (the depthwise kernel is 3x3)
 *   idx     (host struct, device arrays) outputs, capacity >= N*H*W
 *   ws      (device) dynconv_indices_workspace_bytes(s) bytes of scratch
 */
dynconv_status dynconv_build_indices(const uint8_t *mask, dynconv_shape s, int32_t dilate,
                                     const dynconv_indices *idx, void *ws, size_t ws_bytes,
                                     void *stream);

/* Workspace bytes that dynconv_block_forward needs. */
size_t dynconv_block_workspace_bytes(dynconv_shape s, const dynconv_block *blk,
                                     dynconv_dtype dt);

/*
 * One gated residual block (Eq. 3 with r = identity), executed on the
 * gathered rows only (Sec. 3.2):
 *   y[i] = x[i] + F(x)[i]  where the mask is active, y[i] = x[i] elsewhere,
 * with F = project(act_dw(DW3x3(act_expand(expand(x))))).  The expansion runs
 * on the dilated positions, the depthwise and projection on the active ones.
 *   x    (device) NHWC input, shape s, dtype dt
 *   y    (device) NHWC output; y == x runs in place, any other overlap is
 *        DYNCONV_ERR_SHAPE; when y != x inactive positions are copied
 *   blk  (host struct, device weights)
 *   idx  (host struct, device arrays) built by dynconv_build_indices with
 *        dilate >= 1, or NULL for the dense block (Eq. 1) on all positions
 *   ws   (device) dynconv_block_workspace_bytes bytes of scratch
 */
dynconv_status dynconv_block_forward(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                     const dynconv_block *blk, const dynconv_indices *idx,
                                     void *ws, size_t ws_bytes, void *stream);

/* Flags of dynconv_stack_forward. */
#define DYNCONV_STACK_DENSE 1   /* every block on all positions (Eq. 1), no mask units */
#define DYNCONV_STACK_UNFUSED 2 /* force the multi-kernel chain (mask, index maps, block) */
#define DYNCONV_STACK_GSOFTMAX 4 /* mask units decide as dynconv_mask_gsoftmax (Sec. 3.1.2) */

/* Workspace bytes that dynconv_stack_forward needs for these blocks and flags. */
size_t dynconv_stack_workspace_bytes(dynconv_shape s, const dynconv_block *blks,
                                     int32_t n_blocks, dynconv_dtype dt, int32_t flags);

/*
 * A stack of gated blocks (Sec. 3.1.1: every residual block has its own mask
 * unit, applied to that block's input), one stream, no host synchronisation.
 * The result is that of
 *   x_0 = x
 *   for b in 0..n_blocks-1:
 *     mask_b  = dynconv_mask(x_b, blks[b].w_mask, blks[b].b_mask)
 *     idx_b   = dynconv_build_indices(mask_b, dilate = 1)
 *     x_{b+1} = dynconv_block_forward(x_b, blks[b], idx_b)
 *   y = x_{n_blocks}
 * With DYNCONV_STACK_DENSE the mask units are skipped and every block runs on
 * all positions (the baseline of Eq. 1).
 *
 * Execution: when s.c <= 64 (fp32) or s.c <= 128 (fp16, bf16) and
 * DYNCONV_STACK_UNFUSED is not set, each
 * block is ONE kernel over small patches of the image (at most 256
 * positions, at most 32 columns wide), each of which builds the active and
 * halo lists of its patch on chip (ballot ranks in raster order), gathers,
 * expands, runs the depthwise and the projection, adds the identity path and
 * computes the next block's mask (the first block also runs its own mask
 * unit); blocks alternate between y and a workspace copy.  The per-block
 * counts P, P_d take one more small kernel, launched only when counts is not
 * NULL.  Otherwise the block runs the kernel chain of the per-block calls,
 * in place on y.  Both give identical masks, counts and outputs: the same
 * arithmetic in the same order.
 *   x      (device) NHWC input, shape s, dtype dt; read only unless y == x
 *   y      (device) NHWC output; y == x runs in place, other overlap is
 *          DYNCONV_ERR_SHAPE
 *   blks   (host array of n_blocks, device weights), 1 <= n_blocks <= 1024
 *   flags  0 or DYNCONV_STACK_DENSE / DYNCONV_STACK_UNFUSED / DYNCONV_STACK_GSOFTMAX
 *          (others: ERR_ARG)
 *   masks  (device) uint8 [n_blocks][N*H*W] or NULL: per-block hard masks
 *   counts (device) int32 [n_blocks][2] or NULL: per-block P, P_d
 *   ws     (device) dynconv_stack_workspace_bytes bytes of scratch
 */
dynconv_status dynconv_stack_forward(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                     const dynconv_block *blks, int32_t n_blocks, int32_t flags,
                                     uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                     void *stream);

/*
 * Launch sequence of dynconv_stack_forward, for profiling: stores up to `cap`
 * kernel names (static strings) in launch order into `names` (may be NULL
 * when cap is 0) and returns the number of launches, or -1 for invalid
 * arguments.  in_place says whether the call will have y == x.  The count
 * reduction (k_band_counts, last) is listed as if counts were requested; a
 * call without counts skips it and leaves its event pair unused.
 */
int32_t dynconv_stack_launch_names(dynconv_shape s, const dynconv_block *blks, int32_t n_blocks,
                                   dynconv_dtype dt, int32_t flags, int32_t in_place,
                                   const char **names, int32_t cap);

/*
 * dynconv_stack_forward with per-kernel timing: launch i of the sequence that
 * dynconv_stack_launch_names reports is issued with the event pair
 * (events[2i], events[2i+1]) (hipEvent_t, created by the caller), which the
 * runtime stamps when that kernel starts and ends, so
 * hipEventElapsedTime(events[2i], events[2i+1]) is the kernel's duration.
 * n_events must be at least 2 * count (else DYNCONV_ERR_ARG).  Results are
 * identical to dynconv_stack_forward.
 */
dynconv_status dynconv_stack_forward_profiled(const void *x, void *y, dynconv_shape s,
                                              dynconv_dtype dt, const dynconv_block *blks,
                                              int32_t n_blocks, int32_t flags, uint8_t *masks,
                                              int32_t *counts, void *ws, size_t ws_bytes,
                                              void *stream, void *const *events,
                                              int32_t n_events);

/*
 * dynconv_stack_forward for callers that cannot allocate device memory:
 * code under HIP graph capture that must not call hipMalloc, tight serving
 * loops, harnesses that forbid allocation.  It takes no workspace: the
 * library keeps one static scratch array of
 * dynconv_stack_noalloc_max_workspace_bytes() (16 MiB) in device memory on
 * every device it runs on, held until the process ends, and this call uses
 * the current device's copy.  Arguments, results and errors are those of
 * dynconv_stack_forward (the same kernels, bit-identical output), except:
 *   * a stack whose dynconv_stack_workspace_bytes exceeds the array returns
 *     DYNCONV_ERR_WORKSPACE and enqueues nothing;
 *   * the first call on a device looks the array up (hipGetSymbolAddress;
 *     a failure returns DYNCONV_ERR_HIP);
 *   * it calls no hipMalloc, hipFree or other allocating routine.
 * Every call on one device shares that device's array and leaves the last
 * call's contents in it (nothing in it needs to start at zero), so calls
 * that overlap in time on one device race: serialise them (one stream, or
 * events between streams).
 */
size_t dynconv_stack_noalloc_max_workspace_bytes(void);
dynconv_status dynconv_stack_forward_noalloc(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                             const dynconv_block *blks, int32_t n_blocks, int32_t flags,
                                             uint8_t *masks, int32_t *counts, void *stream);

/*
 * ShuffleNetV2 stride-1 units whose convolutional branch is a gated residual
 * block (Sec. 4.1.2: dynamic convolutions in the branch of the non-strided
 * units of ShuffleNetV2 with a residual connection; the branch is Eq. 3 with
 * r = identity).  With cb = s.c / 2, unit u maps its input x_u to
 *   x1 = x_u[..., 0 .. cb-1],  x2 = x_u[..., cb .. 2cb-1]
 *   mask_u = dynconv_mask(x2 zero-extended to cp channels, branches[u].w_mask,
 *                         branches[u].b_mask)
 *   b  = x2 + F(x2) where mask_u is 1, b = x2 elsewhere, with F the branch
 *        block (expand, depthwise 3x3, project with its activations;
 *        ShuffleNetV2: RELU, NONE, RELU) on x2 zero-extended to cp channels,
 *        of which the first cb outputs are kept
 *   x_{u+1}[..., 2k] = x1[k],  x_{u+1}[..., 2k+1] = b[k]    (k < cb)
 * i.e. channel_shuffle(concat(x1, b), 2), and y = x_{n_units}.
 * cp = branches[u].c_in, the same for every unit, with cb <= cp, cp a
 * multiple of 8 (so cb = 58 runs as cp = 64); the branch weights act on cp
 * channels (the caller zero-pads PyTorch's cb-channel weights; since the
 * padded input channels are zero, their weight columns do not matter, and
 * outputs cb .. cp-1 are discarded).  c_hidden is a multiple of 16 (pad
 * with zero weights).  Execution: when cp fits the one-launch block kernel
 * (cp <= 64 in fp32, cp <= 128 in fp16/bf16), cb * sizeof(dtype) is a
 * multiple of 4 and DYNCONV_STACK_UNFUSED is not set, each unit is ONE
 * launch on the unit's own rows: it stages the branch half (zero-extended
 * to cp channels) and the pass-through half, runs the gated block and
 * writes the shuffled rows.  Otherwise the branch input is copied into
 * compact cp-channel rows, the branch runs as one gated block (the
 * one-launch kernel or the kernel chain), and one kernel writes the
 * shuffled unit output together with the next unit's branch rows.
 *   x, y   (device) NHWC, shape s (s.c even), dtype dt; must not overlap
 *   branches (host array of n_units, device weights), 1 <= n_units <= 1024
 *   flags  0 or DYNCONV_STACK_DENSE (every branch on all positions, no mask
 *          units) / DYNCONV_STACK_UNFUSED / DYNCONV_STACK_GSOFTMAX; others: ERR_ARG
 *   masks  (device) uint8 [n_units][N*H*W] or NULL: per-unit hard masks
 *   counts (device) int32 [n_units][2] or NULL: per-unit P, P_d
 *   ws     (device) dynconv_shuffle_stack_workspace_bytes bytes of scratch
 * Errors as for dynconv_stack_forward; an odd s.c, cp < cb, or branch
 * blocks of different c_in are DYNCONV_ERR_SHAPE.
 */
size_t dynconv_shuffle_stack_workspace_bytes(dynconv_shape s, const dynconv_block *branches,
                                             int32_t n_units, dynconv_dtype dt, int32_t flags);

dynconv_status dynconv_shuffle_stack_forward(const void *x, void *y, dynconv_shape s, dynconv_dtype dt,
                                             const dynconv_block *branches, int32_t n_units,
                                             int32_t flags, uint8_t *masks, int32_t *counts, void *ws,
                                             size_t ws_bytes, void *stream);

/* Launch sequence of dynconv_shuffle_stack_forward (as for
 * dynconv_stack_launch_names; k_band_counts, when listed, is last). */
int32_t dynconv_shuffle_stack_launch_names(dynconv_shape s, const dynconv_block *branches,
                                           int32_t n_units, dynconv_dtype dt, int32_t flags,
                                           const char **names, int32_t cap);

/* dynconv_shuffle_stack_forward with per-kernel event pairs, as
 * dynconv_stack_forward_profiled. */
dynconv_status dynconv_shuffle_stack_forward_profiled(const void *x, void *y, dynconv_shape s,
                                                      dynconv_dtype dt, const dynconv_block *branches,
                                                      int32_t n_units, int32_t flags, uint8_t *masks,
                                                      int32_t *counts, void *ws, size_t ws_bytes,
                                                      void *stream, void *const *events,
                                                      int32_t n_events);

/*
 * Whole networks: a MobileNetV2 feature extractor whose stride-1 residual
 * blocks are gated (Sec. 3.1.1: every residual block gets its own mask unit;
 * Sec. 4.1.2: dynamic convolutions in MobileNetV2, with the stem, the strided
 * and the width-changing blocks evaluated at every position).
 */
typedef enum {
    DYNCONV_LAYER_CONV3X3 = 0, /* full 3x3 convolution, zero padding 1 (the stem) */
    DYNCONV_LAYER_BLOCK = 1,   /* inverted-residual block */
    DYNCONV_LAYER_CONV1X1 = 2  /* pointwise convolution */
} dynconv_layer_kind;

/*
 * One layer (host struct, device weights; PyTorch layouts in the storage
 * dtype, fp32 biases):
 *   CONV3X3  w [c_out][c_in][3][3], b [c_out], act, stride 1 or 2;
 *            y[o][i][j] = act(sum w[o][c][kh][kw] x[c][s*i+kh-1][s*j+kw-1] + b[o]),
 *            output (H-1)/stride+1 x (W-1)/stride+1; 1 <= c_in <= 16,
 *            c_out a multiple of 8, 9*c_in*c_out + c_out <= 16384
 *   CONV1X1  w [c_out][c_in], b [c_out], act; c_in, c_out multiples of 8,
 *            c_out <= 4096
 *   BLOCK    blk: expansion 1x1 (w_expand NULL for an expansion factor of 1,
 *            then c_hidden = c_in), depthwise 3x3 with `stride`, projection
 *            1x1, each with its activation; the block adds its input when
 *            stride is 1 and c_in == c_out (Eq. 1, r = identity).
 *            gated = 1 (stride 1, c_in == c_out, w_expand present): the gated
 *            block of Eq. 3 with blk's mask unit, executed as
 *            dynconv_stack_forward executes one block (constraints of
 *            dynconv_block apply); gated = 0: every position, channel
 *            counts multiples of 8, c_hidden <= 1792 (the depthwise weights
 *            are staged in 64 KB of LDS), c_out <= 4096.
 * c_in/c_out of BLOCK layers are blk.c_in/blk.c_out; the layer's own c_in,
 * c_out, w, b, act are for the convolutions.
 */
typedef struct {
    int32_t kind;
    int32_t stride;
    int32_t gated;
    int32_t c_in, c_out;
    const void *w;
    const float *b;
    int32_t act;
    dynconv_block blk;
} dynconv_layer;

/* Output shape of a layer list applied to `in` (its c = the first layer's
 * c_in); errors as dynconv_network_forward's validation. */
dynconv_status dynconv_network_output_shape(dynconv_shape in, const dynconv_layer *layers, int32_t n_layers,
                                            dynconv_shape *out);

/* Workspace bytes of dynconv_network_forward (0 for invalid arguments). */
size_t dynconv_network_workspace_bytes(dynconv_shape in, const dynconv_layer *layers, int32_t n_layers,
                                       dynconv_dtype dt, int32_t flags);

/*
 * y = layers(x), one stream, no host synchronisation.
 *   x      (device) NHWC input, shape `in`, dtype dt
 *   y      (device) NHWC output of dynconv_network_output_shape; must not
 *          overlap x
 *   layers (host array of n_layers, device weights), 1 <= n_layers <= 1024
 *   flags  0 / DYNCONV_STACK_DENSE (gated blocks on every position, no mask
 *          units) / DYNCONV_STACK_UNFUSED / DYNCONV_STACK_GSOFTMAX (as for
 *          dynconv_stack_forward; others: ERR_ARG)
 *   masks  (device) uint8 or NULL: the hard masks of the gated blocks in
 *          layer order, each N*H*W of that block's resolution, concatenated
 *   counts (device) int32 [number of gated blocks][2] or NULL: P, P_d
 *   ws     (device) dynconv_network_workspace_bytes bytes of scratch
 * Every layer is validated before anything is enqueued (ERR_SHAPE for a
 * width that does not chain, ERR_UNSUPPORTED for widths the kernels do not
 * take, ERR_ARG for a bad kind, stride or activation).
 */
dynconv_status dynconv_network_forward(const void *x, void *y, dynconv_shape in, dynconv_dtype dt,
                                       const dynconv_layer *layers, int32_t n_layers, int32_t flags,
                                       uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                       void *stream);

/* Launch sequence of dynconv_network_forward, as dynconv_stack_launch_names;
 * with_counts says whether the call will pass counts (each gated block then
 * ends with its count reduction). */
int32_t dynconv_network_launch_names(dynconv_shape in, const dynconv_layer *layers, int32_t n_layers,
                                     dynconv_dtype dt, int32_t flags, int32_t with_counts, const char **names,
                                     int32_t cap);

/* dynconv_network_forward with per-kernel event pairs, as
 * dynconv_stack_forward_profiled. */
dynconv_status dynconv_network_forward_profiled(const void *x, void *y, dynconv_shape in, dynconv_dtype dt,
                                                const dynconv_layer *layers, int32_t n_layers, int32_t flags,
                                                uint8_t *masks, int32_t *counts, void *ws, size_t ws_bytes,
                                                void *stream, void *const *events, int32_t n_events);

#ifdef __cplusplus
}
#endif

#endif /* DYNCONV_H_ */
