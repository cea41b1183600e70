// Internal declarations shared by the host planner (api.hip) and the kernels.
//
// Data layout of every layer's activations ("fragment batch"):
//   [B * F][Hmax][Wmax][C], channels innermost,
// where F is the number of fragments per image at that layer, Hmax x Wmax the
// largest fragment size, and the fragment of image b with per-axis indices
// (fy, fx) sits at batch index b * F + fy * Qx + fx (Qy, Qx = products of the
// pools' row and column sizes so far, F = Qy * Qx; square pools give
// Qy = Qx).  Fragment sizes are separable: a fragment's height
// depends only on its y-offset chain and its width only on its x-offset chain,
// so one table per axis (indexed by fy or fx) holds every fragment's true
// size.  Pixels beyond a fragment's true size are padding: never read for a
// valid output and never written.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace fs {

constexpr int kMaxAxis = 256;   // per-axis fragment count limit (product of pool sizes)
constexpr int kMaxSide = 65535; // image rows / columns of one scan (fragment sizes are 16-bit)
constexpr int kMaxHeadClasses = 16;
// Head kernel: kHeadLanesPerPixel lanes share one output pixel's channel
// vector, and each group of them takes kHeadPixelsPerGroup pixels in turn, so
// a workgroup's weight staging serves 256 / kHeadLanesPerPixel *
// kHeadPixelsPerGroup pixels.
constexpr int kHeadLanesPerPixel = 4;
constexpr int kHeadPixelsPerGroup = 4;
constexpr int kMaxHeadWeights = 8192;  // n_classes * c_in of a fused last layer
constexpr size_t kMaxLdsBytes = 160 * 1024;  // LDS of one CDNA4 compute unit
constexpr int kMaxChannels = 16384;           // per layer (kernels divide by channel counts below 2^16)
constexpr int kMaxFusedClasses = 4;   // classes of a last layer fused into a conv epilogue

// Bounds checks (debug builds: compiled with -DFRAGSCAN_DEBUG into
// libfragscan_debug.so).  Every fragment read and write of the kernels is
// checked against the true size of its fragment (the per-axis tables, or
// Eqs. 6-7 for a pool's children) and its buffer's batch and row pitch, every
// output-map write against the map.  A failed check sets bit `site` of the
// launch's status word (`dbg`, device memory the host clears before a scan
// and reads after it) and skips the access, so the kernel still ends
// normally; the scan then returns FS_ERR_BOUNDS naming the sites.  A launch's
// `dbg_shrink` (0 unless forced from the host to test that path) is taken
// off every true size the checks use.  Release builds compile the checks out.
enum DbgSite {
    DBG_CONV_READ = 0,     // convolution: input window
    DBG_CONV_WEIGHT = 1,   // convolution: weight / bias blocks of the tile
    DBG_CONV_WRITE = 2,    // convolution: output fragment
    DBG_FUSED_POOL = 3,    // convolution + pool: child fragment
    DBG_FUSED_HEAD = 4,    // convolution + last layer: output map
    DBG_POOL_READ = 5,     // pool: parent fragment
    DBG_POOL_WRITE = 6,    // pool: child fragment
    DBG_HEAD_READ = 7,     // head: final fragment
    DBG_HEAD_WRITE = 8,    // head: output map
    DBG_PAD_READ = 9,      // mirror pad: image
    DBG_NSITES = 10
};
#ifdef FRAGSCAN_DEBUG
__device__ __forceinline__ bool dbg_check(unsigned *word, bool ok, int site)
{
    if (!ok) atomicOr(word, 1u << site);
    return ok;
}
#define FS_DBG_OK(word, cond, site) ::fs::dbg_check((word), (cond), (site))
#else
#define FS_DBG_OK(word, cond, site) true
#endif

enum ActKind { ACT_NONE = 0, ACT_TANH = 1, ACT_SOFTMAX = 2 };
enum DType { DT_F32 = 0, DT_BF16 = 1 };

// Per-axis true sizes of the fragments a launch reads.
struct AxisTable {
    uint16_t y[kMaxAxis];
    uint16_t x[kMaxAxis];
};

// Fragment-batched convolution (also the fully connected layers, as
// convolutions with k = size of the map they receive).
struct ConvArgs {
    const void *in;       // [nfrag][in_h][in_w][in_c] (float or bf16; first layer: the image)
    void *out;            // [nfrag][out_h][out_w][cout]
    const void *w;        // packed weights (api.hip: pack_conv_weights)
    const float *bias;    // [nbt * 16] in (block, row) order, zero padded
    int nfrag;            // B * F
    int F, Qy, Qx;        // fragments per image, per axis
    int in_h, in_w, in_c; // padded input dims; in_c = channel pitch of the input
    int out_h, out_w;     // padded output dims
    int ky, kx, cin, cout, act;  // kernel rows, columns
    int ksteps;           // K steps of the matrix-core loop
    int nbt;              // total 16-wide output-channel blocks
    int nbu;              // blocks holding output channels (ceil(cout / 16)); past them the register tile pads
    int swapn;            // 1: channel halves swapped between the two wave columns in alternate workgroups
    int band_w;           // output columns per band
    int nbands;           // bands per fragment
    int tiles_per_band;   // tiles per band (enough for the tallest fragment)
    int mt;               // output pixels per tile (16 * MB * 4 / (WN * WK))
    int tile_rows;        // > 0: a tile is tile_rows whole rows of its band (tile_rows * band_w <= mt)
    int lds_cs;           // channel stride of a pixel in LDS (elements)
    int lds_bytes;        // dynamic LDS bytes of one workgroup
    int direct_store;     // 1: lanes store their channel runs straight to memory;
                          // 0: restaged through LDS and written as whole rows
    // Fused max-pool (pool_k > 0): the launch also applies the k x k pool that
    // follows the convolution and writes its children straight to `out`
    // ([nfrag * k^2][pool_oh][pool_ow][cout]); bands then run over the
    // stride-1 max filter's columns, and a tile is pool_rt filter rows plus
    // the k - 1 rows and columns of convolution outputs they also need.
    int pool_ky, pool_kx, pool_rt, pool_oh, pool_ow;  // pool_ky == 0: no pool
    // Run tiles (run > 0; layers whose fragments each fit one band and hold
    // at least mt output pixels): per image the fragments' output pixels are
    // numbered in fragment order, fragment (fy, fx) holding
    // [ypre[fy] * wsum + ho[fy] * xpre[fx], ... + ho[fy] * wo[fx]) with ho, wo
    // its output sizes and ypre / xpre their per-axis prefix sums (wsum =
    // xpre[Q]); a tile is mt consecutive pixels of that sequence, so it may
    // end in one fragment and continue in the next.  tiles_per_band is then
    // tiles per image.
    int run, run_pix, run_wsum;
    uint16_t run_ypre[kMaxAxis + 1], run_xpre[kMaxAxis + 1];
    AxisTable ext;        // true sizes of the input fragments
    // Fused last layer (head_ncls > 0): the 1x1 layer cout -> head_ncls, its
    // activation, and the reassembly are applied in the epilogue, which then
    // writes the dense output map instead of `out`'s fragment batch.
    int head_ncls, head_act;
    // xsib = 1 (fused head, fragment tiles): tiles are numbered with the
    // fragment's column index fx fastest, so the Qx fragments of one row of
    // the grid, whose outputs interleave in the map's columns (column
    // base_x[fx] + Sx * x), run the same tile side by side and fill the map's
    // memory lines together.
    int xsib;
    const float *head_w;  // [max(head_ncls, kMaxFusedClasses)][nbt * 16], columns in (block, row) order, zero rows past head_ncls
    // bf16 nets whose tile pairs channel blocks: the same weights as the row
    // operand of a 16x16x32 bf16 product, [nbt / 2][64 lanes][8 bf16], lane l
    // holding class l % 16 (zero past head_ncls) at channels
    // 32 * pair + 8 * (l / 16) .. + 7 (zero past the channels)
    const void *head_wbf;
    const float *head_b;  // [head_ncls]
    float *head_out;      // [B][ny][nx][head_ncls] (ny, nx: the output map's rows and row pitch)
    int ny, nx, Sy, Sx;       // Sy, Sx: products of the pools' row / column sizes
    uint16_t base_y[kMaxAxis], base_x[kMaxAxis];  // per-axis fragment index -> its first output coordinate
    unsigned *dbg;            // debug builds: status word of the bounds checks
    int dbg_shrink;
};
// Passed by value: the launch arguments of one dispatch (4 KiB at most).
static_assert(sizeof(ConvArgs) <= 4096, "ConvArgs must stay within the kernel-argument limit");

struct PoolArgs {
    const void *in;      // parents  [B*F][in_h][in_w][C]
    void *out;           // children [B*F*sy*sx][out_h][out_w][C]
    int F, Qx;           // parents per image; per row of the fragment grid
    int in_h, in_w;
    int out_h, out_w;
    int C, ky, kx;       // pool rows, columns
    int sy, sx;          // step between windows, rows and columns (the paper's pools: ky, kx)
    int n_children;      // B * F * sy * sx
    int rows;            // row-band kernel: filter rows per thread (4 or 8)
    AxisTable ext;       // true sizes of the parents
    unsigned *dbg;       // debug builds: status word of the bounds checks
    int dbg_shrink;
};

// Last stage: (optionally) the last 1x1 layer, its activation, and the
// reassembly of final fragments into the dense output map.
struct HeadArgs {
    const void *in;      // final fragments [B*F][in_h][in_w][C]
    float *out;          // [B][out_ny][out_nx][ncls], windows at [.][0, ny)[0, nx)
    const float *w;      // [ncls][C] (has_fc) or unused
    const float *bias;   // [ncls]
    int B, F, Qx;
    int in_h, in_w, C;
    int ny, nx, ncls, act;  // windows per image (rows, columns)
    int out_ny, out_nx;  // the output map's rows and row pitch (>= ny, nx)
    int Sy, Sx;          // products of the pools' row / column sizes
    uint16_t digit_y[kMaxAxis], digit_x[kMaxAxis];  // output coordinate mod S -> per-axis fragment index
    AxisTable ext;       // true sizes of the final fragments (for the bounds checks)
    unsigned *dbg;       // debug builds: status word of the bounds checks
    int dbg_shrink;
};

// Launchers (return hipSuccess or the launch error).  `dtype` selects the
// operand type; `in_f32` says the input is float32 even in a bf16 net (the
// image).  Convolution register tiles: mb pixel blocks x nb channel blocks per
// wave, wn waves across the output channels, wk waves splitting the K steps,
// 4 / (wn * wk) across the pixels.  a.run picks the run-tile instance.
hipError_t launch_conv(const ConvArgs &a, int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec,
                       int grid_x, int grid_y, hipStream_t s);
hipError_t launch_pool(const PoolArgs &a, int dtype, bool in_f32, int grid, hipStream_t s);
// Mirrored borders: out[B][He][We][C] from in[B][H][W][C], extended index
// (y, x) reading image pixel (mirror(y - p0y, H), mirror(x - p0x, W)).
enum BorderMode { BORDER_VALID = 0, BORDER_REFLECT = 1, BORDER_SYMMETRIC = 2 };
hipError_t launch_mirror_pad(const float *in, float *out, int B, int H, int W, int C, int p0y, int p0x, int He,
                             int We, int mode, unsigned *dbg, int dbg_shrink, hipStream_t s);
hipError_t launch_head(const HeadArgs &a, int dtype, bool in_f32, bool has_fc, int grid,
                       hipStream_t s);
// The float32 4 x 13 x 1 x 1 vector-path tile (conv_f32_wide.hip; no run
// tiles, one workgroup per CU); launch_conv routes that shape there.
hipError_t launch_conv_f32_wide(const ConvArgs &a, int gx, int gy, hipStream_t s);
// Whether a tile shape has an instance (run: one with run tiles).
bool conv_tile_supported(int mb, int nb, int wn, int wk, bool vec, bool run = false);
// Workgroups of that convolution kernel resident per CU with `lds` bytes of
// dynamic LDS, on the current device (0 if the query fails).
int conv_blocks_per_cu(int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec, bool run, int lds);
// Direct (vector-ALU) convolution for tiny K = c_in * taps (taps = k_y * k_x,
// K <= 64) and c_out <= 48; wpk = weights as [rows][KP] float32 with rows =
// c_out rounded up to 8 (zero rows past c_out), K index (dy * k_x + dx) *
// c_in + ci, zero padded to KP = conv_direct_kp(c_in, taps) (bf16 nets: values
// rounded to bf16), followed by the c_out biases in channel order.  One thread
// per pixel.
bool conv_direct_supported(int cin, int taps, int cout);
int conv_direct_kp(int cin, int taps);
hipError_t launch_conv_direct(const ConvArgs &a, const float *wpk, int dtype, bool in_f32, int grid, hipStream_t s);
std::string conv_direct_kernel_name(int dtype, bool in_f32, int cin, int taps);

// Kernel names as the profiler reports them (for measurement reports).
std::string conv_kernel_name(int dtype, bool in_f32, int mb, int nb, int wn, int wk, bool vec, bool run);
std::string pool_kernel_name(int dtype, bool in_f32, int ky, int kx, int sy, int sx, int C, int rows);
const char *head_kernel_name(int dtype, bool in_f32, bool has_fc);

}  // namespace fs
