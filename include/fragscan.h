/*
 * fragscan — fragment-based image scanning with deep max-pooling CNNs on
 * AMD Instinct MI355X (gfx950).
 *
 * The library applies a net made of convolutional, max-pooling and fully
 * connected layers to every w_0 x w_0 window of an image in one pass, the way
 * Giusti et al., "Fast Image Scanning with Deep Max-Pooling Convolutional
 * Neural Networks" (IDSIA-01-13) describe in Section 2.2: every convolution is
 * computed once on whole extended maps, every k x k max-pooling layer splits
 * each fragment into k^2 fragments, one per pooling offset, and the fragments
 * of the last layer are put back together into a dense map holding, for every
 * window, the net's output (class posterior probabilities when the last layer
 * is a softmax, Section 1).
 *
 * Conventions used throughout
 *   - A window ("patch") is named by its top-left pixel (Y, X); the output
 *     map has (H - w_0 + 1) x (W - w_0 + 1) entries per image (Section 2.2:
 *     all windows completely contained in the image).
 *   - Images are [B][H][W][C] float32, channels innermost; outputs are
 *     [B][H - w_0 + 1][W - w_0 + 1][n_classes] float32.
 *   - Convolutions are valid cross-correlations; weights are OIHW
 *     [c_out][c_in][k][k] float32, biases [c_out] float32.
 *   - Fragment ids follow the offset order of Section 2.2.2 (o_x fastest):
 *     the child of fragment f at pooling offset (o_x, o_y) of a k x k pool is
 *     f * k^2 + o_y * k + o_x, starting from fragment 0 (the whole image).
 *   - Rectangular kernels, pools and windows (Section 2: the square case
 *     generalises directly): a layer's k_x gives its columns, the window is
 *     h_0 x w_0, and every rule above holds per axis, rows with h_0 and k,
 *     columns with w_0 and k_x (a k x k_x pool has k * k_x children).
 *   - Pools whose windows step by s instead of their size k (overlapping for
 *     s < k, leaving gaps for s > k; not in the paper, whose pools do not
 *     overlap): the patch-level map side w becomes (w - k) / s + 1 and must
 *     divide exactly, and every rule above holds with s in place of k where
 *     it counts children and offsets: s^2 children f * s^2 + o_y * s + o_x,
 *     o in {0..s-1}^2, each holding div(n - o - k + s, s) pixels per axis of
 *     a parent of n (the windows starting at o, o + s, ... that end inside
 *     it).
 *
 * Errors: every call returns an fs_status and never throws or aborts across
 * this boundary; fs_last_error() gives a thread-local message for the last
 * failing call on the calling thread.  Arguments are validated before any
 * work is enqueued, so a failing fs_scan leaves the stream untouched.
 *
 * Memory: pointers named d_* are device pointers (HIP device memory the caller
 * owns); pointers named h_* or described as host are host memory.  A net owns
 * the device copy of its weights from fs_net_create to fs_net_destroy.
 */
#ifndef FRAGSCAN_H
#define FRAGSCAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fs_net fs_net; /* opaque; immutable after fs_net_create */

typedef enum {
    FS_OK = 0,
    FS_ERR_INVALID_ARG = 1,  /* null / misaligned pointer, bad enum, bad count */
    FS_ERR_SHAPE = 2,        /* net or image sizes the method does not allow */
    FS_ERR_UNSUPPORTED = 3,  /* allowed by the method, not by this library */
    FS_ERR_WORKSPACE = 4,    /* workspace smaller than fs_scan_plan asks for */
    FS_ERR_OOM = 5,          /* device allocation failed (fs_net_create only) */
    FS_ERR_HIP = 6,          /* a HIP runtime call failed */
    FS_ERR_BOUNDS = 7        /* debug library only (libfragscan_debug.so): a kernel's
                              * bounds check failed; fs_last_error names the checks.
                              * The scan skipped those accesses: its output is not valid.
                              * Its scans synchronise their stream, and scans that overlap
                              * on one device share one status word (a failure may be
                              * reported by any of them) */
} fs_status;

/* Layer kinds (Section 2: input, convolutional, max-pooling and fully
 * connected layers).  A fully connected layer is applied to every fragment
 * as a convolution whose kernel covers the whole patch-level map it receives
 * (k = w_L for the first one, then 1); a fragment at any layer depends on one
 * fragment of the layer below (Section 3). */
typedef enum { FS_CONV = 0, FS_MAXPOOL = 1, FS_FC = 2 } fs_kind;

/* Activation after a layer.  FS_ACT_SOFTMAX is allowed on the last layer only
 * and turns its outputs into class posterior probabilities (Section 1). */
typedef enum { FS_ACT_NONE = 0, FS_ACT_TANH = 1, FS_ACT_SOFTMAX = 2 } fs_act;

/* Storage and matrix-core operand type of activations and weights.  FS_BF16
 * rounds the image, weights and every stored activation to bfloat16 (round to
 * nearest even) and accumulates, adds biases, applies activations and the
 * softmax in float32. */
typedef enum { FS_F32 = 0, FS_BF16 = 1 } fs_dtype;

/* One layer.  For FS_MAXPOOL: k = pool size, c_in = c_out = channels, weight
 * and bias NULL, act FS_ACT_NONE.  For FS_CONV / FS_FC: k = kernel size
 * (FS_FC may pass 0 to take the size of the map it receives), weight = host
 * OIHW [c_out][c_in][k][k_x] float32, bias = host [c_out] float32 or NULL for
 * zeros.  Host arrays are copied by fs_net_create and not kept.
 * k_x: the kernel's or pool's columns when they differ from its rows k
 * (Section 2: the square case generalises directly to rectangles, each rule
 * holding per axis); 0 means k_x = k.  An FS_FC layer passing k = 0 passes
 * k_x = 0 too.
 * stride, stride_x (FS_MAXPOOL only): rows / columns between the starts of
 * neighbouring pooling windows; stride 0 means k (the paper's
 * non-overlapping pools), stride_x 0 means stride when stride is given, else
 * k_x.  Convolutions and fully connected layers pass 0 (stride 1; any other
 * value gives FS_ERR_UNSUPPORTED). */
typedef struct {
    int32_t kind;
    int32_t k;
    int32_t c_in;
    int32_t c_out;
    int32_t act;
    const float *weight;
    const float *bias;
    int32_t k_x;
    int32_t stride;
    int32_t stride_x;
} fs_layer;

typedef struct {
    int32_t patch;        /* w_0 (rectangular windows: h_0, the rows) */
    int32_t in_channels;  /* C */
    int32_t n_classes;    /* c_out of the last layer */
    int32_t n_layers;
    int32_t n_pools;
    int32_t stride;       /* product of the pools' strides (their sizes for the
                             paper's pools): output pixels one final fragment
                             pixel step covers, per axis (rows) */
    int32_t n_fragments;  /* F_L, the product of the squared pool sizes
                             (Section 3; rectangular pools: of k * k_x;
                             strided pools: of stride * stride_x) */
    int32_t dtype;        /* fs_dtype */
    int32_t patch_x;      /* the window's columns (= patch for square nets) */
    int32_t stride_x;     /* product of the pools' column strides (k_x) */
} fs_net_info;

typedef struct {
    int32_t batch;
    int32_t out_h;           /* H - h_0 + 1 (h_0 = w_0 for square windows) */
    int32_t out_w;           /* W - w_0 + 1 */
    int32_t n_launches;      /* kernel launches fs_scan enqueues */
    size_t workspace_bytes;  /* device workspace fs_scan needs */
    double flops;            /* algorithmic FLOPs of one scan: 2 * c_in * k^2 *
                                c_out per output pixel of every fragment of
                                every conv / fc layer */
    double min_bytes;        /* sum over launches of the bytes each must move
                                at least (read its input once, write its output
                                once, read its weights once) */
} fs_plan_info;

/* Per-launch description, for measurement.  `name` is the kernel's symbol-
 * like label as it appears in profiler traces (NUL-terminated). */
typedef struct {
    int32_t layer;        /* first net layer this launch computes */
    int32_t n_layers;     /* net layers it covers (a fused head covers 1-2) */
    int32_t kind;         /* 0 conv, 1 pool, 2 head */
    int32_t fragments;    /* B * fragments written by this launch */
    int64_t out_pixels;   /* true output pixels written, all fragments */
    double flops;         /* algorithmic FLOPs (see fs_plan_info) */
    double bytes;         /* minimum bytes (see fs_plan_info) */
    int32_t grid;         /* workgroups launched */
    int32_t block;        /* threads per workgroup */
    char name[96];
    int32_t lds_bytes;    /* dynamic LDS per workgroup */
    int32_t per_cu;       /* workgroups resident per CU (registers and LDS;
                             0 when unknown, e.g. plan-only nets) */
} fs_launch_info;

/* Create a net.  The stack must be: conv / max-pool layers in any order, then
 * one or more fully connected layers (Section 2); channels must chain; every
 * pool must divide the patch-level map it receives (Section 2.1.2:
 * mod(w_{l-1}, k) = 0; with a stride s, mod(w_{l-1} - k, s) = 0); the
 * patch-level map after the last layer must be 1 x 1.  `patch` is w_0 (0: derive it from the stack; a rectangular stack,
 * whose window is h_0 x w_0 with h_0 != w_0, must pass 0 and give its fully
 * connected sizes).  A patch that does
 * not agree with the stack gives FS_ERR_SHAPE; more than 16384 channels in a
 * layer gives FS_ERR_UNSUPPORTED.  A convolution stages its input window with
 * all of its input channels in the 160 KB of LDS, so planning a scan
 * (fs_scan_plan and the scans) gives FS_ERR_UNSUPPORTED for a layer with more
 * input channels than a minimal window holds: about 150 (float32, 5 x 5
 * kernel), 245 (3 x 3), 320 (2 x 2), 440 (1 x 1); bfloat16 265, 450, 610, 860.
 * Weights are converted (and
 * for FS_BF16 rounded) and uploaded to the current HIP device, which the net
 * is then bound to.  On success *out receives the handle. */
fs_status fs_net_create(const fs_layer *layers, int32_t n_layers, int32_t in_channels,
                        int32_t patch, int32_t dtype, fs_net **out);

/* The same validation and packing as fs_net_create, without touching any
 * device: the handle answers fs_net_query, fs_scan_plan, fs_scan_launches,
 * fs_fragment_table and fs_reassembly_index (host-side planning, e.g. on a
 * machine without a GPU); fs_scan and fs_scan_profile reject it with
 * FS_ERR_INVALID_ARG.  Release it with fs_net_destroy. */
fs_status fs_net_create_plan_only(const fs_layer *layers, int32_t n_layers, int32_t in_channels,
                                  int32_t patch, int32_t dtype, fs_net **out);

/* Release a net and its device memory.  NULL is ignored.  The caller must
 * make sure no scan using the net is still running. */
void fs_net_destroy(fs_net *net);

fs_status fs_net_query(const fs_net *net, fs_net_info *out);

/* Sizes and work of a scan of B images of H x W (Section 2.2: an s x s image
 * with s >= w_0 gives (s - w_0 + 1)^2 windows; rectangular images are the
 * per-axis generalisation).  FS_ERR_SHAPE if H or W < w_0 or B < 1.
 * FS_ERR_UNSUPPORTED if H or W is above 65535 (fragment sizes are kept in
 * 16-bit tables; fs_scan_tiled scans such an image in regions of at most that
 * size), if B times the net's final fragment count reaches 2^24, or if a
 * fragment would hold 2^31 or more elements. */
fs_status fs_scan_plan(const fs_net *net, int32_t B, int32_t H, int32_t W, fs_plan_info *out);

/* Per-launch description of the scan fs_scan would enqueue; writes
 * min(capacity, n_launches) entries. */
fs_status fs_scan_launches(const fs_net *net, int32_t B, int32_t H, int32_t W,
                           fs_launch_info *h_out, int32_t capacity);

/* Scan B images: the fragment-based forward propagation of Section 2.2 (every
 * convolution computed once on the extended maps of every fragment, Eqs. 3-4;
 * every k x k max-pool splitting each fragment into its k^2 offset children,
 * Eqs. 5-7), then the last layer's softmax and the reassembly of the final
 * fragments into one output per window (Section 3: the fragments cover every
 * window exactly once).  Same limits as fs_scan_plan.
 * d_image: device [B][H][W][C] float32, 16-byte aligned; d_out: device
 * [B][H-w_0+1][W-w_0+1][n_classes] float32, 16-byte aligned; d_workspace:
 * device scratch of at least fs_scan_plan's workspace_bytes, 256-byte aligned
 * (contents need not be initialised and are clobbered); the three must not
 * overlap.  FS_ERR_INVALID_ARG for a NULL or misaligned pointer,
 * FS_ERR_WORKSPACE for a workspace below the plan's size.  `stream` is a
 * hipStream_t (NULL = the default stream).  Asynchronous: returns once every
 * kernel is enqueued; a device fault shows up at the caller's next stream
 * synchronisation.  Calls on different streams with distinct workspaces and
 * outputs may run concurrently on one net. */
fs_status fs_scan(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W,
                  float *d_out, void *d_workspace, size_t workspace_bytes, void *stream);

/* Bytes of the per-GPU scratch array that stands in for the workspace of
 * fs_scan_noalloc (128 MiB: net N4 on a 512 x 512 image needs 99 MB). */
#define FS_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/* fs_scan for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): no
 * workspace argument, and the call allocates nothing.  The workspace is a
 * static device array of FS_NOALLOC_SCRATCH_BYTES that every GPU using the
 * library holds until the process ends (its address is looked up when a net
 * is created on that GPU, or at the first call there).  Every call on one GPU
 * shares that array: calls that overlap on one GPU (on two streams, or from
 * two threads) race and give undefined outputs; the caller serialises them.
 * The array keeps the last call's contents, which no scan depends on.
 * FS_ERR_WORKSPACE when fs_scan_plan's workspace_bytes for this scan exceeds
 * FS_NOALLOC_SCRATCH_BYTES (fs_scan then takes a workspace of the caller's);
 * otherwise the arguments, limits and errors of fs_scan. */
fs_status fs_scan_noalloc(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W,
                          float *d_out, void *stream);

/* Border handling (Section 3.2: the image's edges are mirrored so that the
 * net can be applied at every position).  FS_BORDER_VALID is the plain scan
 * above.  The mirrored modes extend the image by p0 = floor((w_0 - 1) / 2)
 * pixels before the first row / column and w_0 - 1 - p0 after the last, so
 * that output (y, x) is the window whose central pixel (for even w_0: the
 * pixel p0 below and right of its top-left) is image pixel (y, x), and the
 * output map is H x W.  Index i outside [0, n) maps to
 *   FS_BORDER_REFLECT:   period 2(n - 1), mirrored about the edge pixels
 *                        (..., 2, 1, | 0, 1, 2, ...), n = 1: pixel 0;
 *   FS_BORDER_SYMMETRIC: period 2n, edge pixels repeated
 *                        (..., 1, 0, | 0, 1, ...),
 * repeatedly for borders wider than the image.  The paper does not say
 * which of the two it used. */
typedef enum {
    FS_BORDER_VALID = 0,
    FS_BORDER_REFLECT = 1,
    FS_BORDER_SYMMETRIC = 2
} fs_border;

/* fs_scan_plan for a border mode: out_h = H and out_w = W for the mirrored
 * modes; workspace_bytes includes the extended image.  FS_ERR_INVALID_ARG
 * for an unknown mode. */
fs_status fs_scan_plan_border(const fs_net *net, int32_t B, int32_t H, int32_t W, int32_t border,
                              fs_plan_info *out);

/* fs_scan for a border mode: d_out is [B][out_h][out_w][n_classes] as
 * fs_scan_plan_border gives it (H x W for the mirrored modes, any H, W >= 1);
 * the extended image is built in d_workspace, which must hold
 * fs_scan_plan_border's workspace_bytes.  Otherwise as fs_scan. */
fs_status fs_scan_border(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W,
                         int32_t border, float *d_out, void *d_workspace, size_t workspace_bytes,
                         void *stream);

/* Tiled scan: the same outputs as fs_scan (bit for bit) with a workspace
 * bounded by the tile instead of the image, for images whose scan would not
 * fit in device memory.  The H - w_0 + 1 by W - w_0 + 1 output map is cut
 * into tiles of at most tile_h x tile_w windows; each tile is an ordinary
 * fragment scan of the image region its windows cover (tile_h + w_0 - 1 rows
 * of the image, read in place with the image's own pitch; Section 2.2 on that
 * region), writing straight into its place in d_out, and the tiles run one
 * after the other on `stream`, reusing d_workspace.  Each tile recomputes
 * the convolutions of the w_0 - 1 image rows and columns it shares with its
 * neighbours.  d_image [B][H][W][C] float32 and d_out [B][H - w_0 + 1]
 * [W - w_0 + 1][n_classes] float32, device, 16-byte aligned; d_workspace
 * 256-byte aligned, holding fs_scan_plan_tiled's workspace_bytes.  The net's
 * first layer must be a convolution (FS_ERR_UNSUPPORTED otherwise);
 * FS_ERR_INVALID_ARG for tile sizes below 1 or more than 2^20 tiles.  Tile
 * sizes above the map's are clamped to it. */
fs_status fs_scan_plan_tiled(const fs_net *net, int32_t B, int32_t H, int32_t W, int32_t tile_h,
                             int32_t tile_w, fs_plan_info *out);
fs_status fs_scan_tiled(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W,
                        int32_t tile_h, int32_t tile_w, float *d_out, void *d_workspace,
                        size_t workspace_bytes, void *stream);

/* fs_scan with every launch repeated `reps` times back to back between two
 * HIP events on `stream` (a repetition recomputes the same values, so d_out
 * ends as after fs_scan); synchronises the stream and writes, per launch,
 * the events' elapsed time / reps in milliseconds (the launch's mean
 * duration) into h_launch_ms[0 .. min(capacity, n_launches)).  For
 * measurement only. */
fs_status fs_scan_profile(const fs_net *net, const float *d_image, int32_t B, int32_t H,
                          int32_t W, float *d_out, void *d_workspace, size_t workspace_bytes,
                          void *stream, int32_t reps, float *h_launch_ms, int32_t capacity);

/* Fragment table of a scan of an H x W image: for every final fragment
 * f = 0 .. F_L - 1 a record of 5 + 2 * n_pools int32:
 *   f, h_f, w_f, Y0, X0, then (o_x, o_y) of each pool in layer order,
 * where (h_f, w_f) is the fragment's size after the last layer (Eqs. 3-4 and
 * 6-7, never below 0) and output pixel (Y0 + stride * y, X0 + stride_x * x)
 * holds the fragment's pixel (y, x).  The children of fragment f of a
 * k x k_x pool are f * k * k_x + o_y * k_x + o_x (of a pool with strides
 * s x s_x: f * s * s_x + o_y * s_x + o_x).  Host output; writes at most `capacity`
 * int32 and stores the number the full table needs in *n_needed (n_needed
 * may be NULL; h_out may be NULL to query the size). */
fs_status fs_fragment_table(const fs_net *net, int32_t H, int32_t W, int32_t *h_out,
                            size_t capacity, size_t *n_needed);

/* Reassembly index of an H x W image: for every output pixel, row-major over
 * (Y, X), the triple (f, y, x): the final fragment and the position in it
 * that holds the window with top-left corner (Y, X) (Section 3: the union of
 * all fragments covers every window).  Host output, same size protocol as
 * fs_fragment_table (3 * (H - h_0 + 1) * (W - w_0 + 1) int32). */
fs_status fs_reassembly_index(const fs_net *net, int32_t H, int32_t W, int32_t *h_out,
                              size_t capacity, size_t *n_needed);

const char *fs_status_str(fs_status s);
const char *fs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FRAGSCAN_H */
