// C-ABI of the fragment scan: net validation, weight packing, the per-scan
// fragment plan, and the launch sequence.  Declarations and the contract of
// every entry point are in include/fragscan.h.
//
// Plan of a scan (Section 2.2), per layer, from F_0 = 1 fragment of size
// H x W (Eqs. 1-2):
//   conv / fc : F unchanged, each size s -> s - (k - 1)           (Eqs. 3-4)
//   k-pool    : F -> k^2 F; the child at offset o of a fragment of size s gets
//               div(s - o, k), never below 0                      (Eqs. 6-7)
// Sizes are separable per axis, so each layer keeps one table of heights
// (indexed by the y-offset chain) and one of widths (x-offset chain).
#include "../../include/fragscan.h"
#include "fs_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

using namespace fs;

// Workspace of fs_scan_noalloc, for callers that cannot allocate device
// memory: one static array in every GPU's copy of this code object, held
// until the process ends.  Host code never uses the name itself (on the host
// it is a stand-in, not a device address): the address each device gives for
// it, from hipGetSymbolAddress, is kept per device below.
static __device__ __align__(256) unsigned char scratch[FS_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

fs_status fail(fs_status s, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

fs_status hip_fail(hipError_t e, const char *what)
{
    return fail(FS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Device address of `scratch` on `device` (which must be current), looked up
// once per device; nullptr with the error set when the lookup fails.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

fs_status scratch_on(int device, void **out)
{
    if (device < 0 || device >= kMaxDevices) return fail(FS_ERR_UNSUPPORTED, "device %d: no scratch slot", device);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (scratch)");
        if (!p || ((uintptr_t)p & 255)) return fail(FS_ERR_HIP, "scratch at %p is not 256-byte aligned", p);
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return FS_OK;
}

#ifdef FRAGSCAN_DEBUG
}  // namespace
// Debug builds: the status word of the kernels' bounds checks (bit i: check
// site i failed), one per device like `scratch`, looked up the same way.
static __device__ __align__(256) unsigned dbg_word[64];
__global__ void dbg_clear(unsigned *w) { w[0] = 0u; }
namespace {
std::mutex g_dbg_mu;
unsigned *g_dbg_ptr[kMaxDevices];

const char *const kDbgSiteName[DBG_NSITES] = {
    "convolution input window", "convolution weight blocks", "convolution output",
    "fused pool child",         "fused head output map",     "pool parent",
    "pool child",               "head fragment",             "head output map",
    "mirror pad image"};
#endif

// The bounds-check status word of this call (debug builds), cleared on
// stream s before the call's launches; nullptr in release builds.
fs_status dbg_begin(hipStream_t s, unsigned **word)
{
    *word = nullptr;
#ifdef FRAGSCAN_DEBUG
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(FS_ERR_UNSUPPORTED, "device %d: no status word", dev);
    {
        std::lock_guard<std::mutex> lock(g_dbg_mu);
        if (!g_dbg_ptr[dev]) {
            void *p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(dbg_word));
            if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (dbg_word)");
            g_dbg_ptr[dev] = static_cast<unsigned *>(p);
        }
        *word = g_dbg_ptr[dev];
    }
    hipLaunchKernelGGL(dbg_clear, dim3(1), dim3(1), 0, s, *word);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "bounds-check status clear");
#else
    (void)s;
#endif
    return FS_OK;
}

// After the call's launches (debug builds): wait for them and report the
// failed checks as FS_ERR_BOUNDS.
fs_status dbg_end(hipStream_t s, unsigned *word)
{
#ifdef FRAGSCAN_DEBUG
    unsigned h = 0;
    hipError_t e = hipMemcpyAsync(&h, word, sizeof h, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "bounds-check status read");
    if (h) {
        std::string sites;
        for (int i = 0; i < DBG_NSITES; ++i)
            if (h & (1u << i)) sites += std::string(sites.empty() ? "" : ", ") + kDbgSiteName[i];
        return fail(FS_ERR_BOUNDS, "bounds check failed: %s", sites.c_str());
    }
#else
    (void)s;
    (void)word;
#endif
    return FS_OK;
}

// Debug builds: FRAGSCAN_DEBUG_SHRINK=<i> makes launch i of a scan's plan
// check against true sizes one smaller than the real ones (=pad: the mirror
// pad), so that its checks fail on accesses that are in fact in bounds (a
// test of the failure path that leaves every access inside the buffers);
// -1 (-2 for the pad) when unset or in release builds.
int dbg_shrink_at()
{
#ifdef FRAGSCAN_DEBUG
    const char *v = getenv("FRAGSCAN_DEBUG_SHRINK");
    if (!v || !*v) return -1;
    if (std::strcmp(v, "pad") == 0) return -2;
    return atoi(v);
#else
    return -1;
#endif
}

uint16_t host_f2bf(float f)
{
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

struct NetLayer {
    int kind, k, cin, cout, act;
    int kx;               // columns of the kernel / pool (k: its rows; Section 2's rectangular case)
    int sy = 1, sx = 1;   // pools: the step between windows, rows and columns (the paper's: k, kx)
    int h_in, h_out, w_in, w_out;  // patch-level map sizes (Sections 2.1.1, 2.1.2)
    // conv launch parameters fixed at creation
    bool vec = false;     // channel-vector path
    int nb = 1;           // output-channel blocks per wave
    int wn = 1;           // waves across output channels
    int wk = 1;           // waves splitting the K steps
    int nbt = 0;          // channel blocks, padded to a multiple of nb * wn
    int ksteps = 0;
    size_t w_off = 0, b_off = 0;  // offsets into the net's device block
    bool has_w32 = false;         // OIHW float32 copy for the direct kernel
    size_t w32_off = 0;
};

}  // namespace

struct PlanCache;  // scan plans of a net, by size (defined with the planner)

struct fs_net {
    std::vector<NetLayer> L;
    int patch = 0, C = 0, dtype = 0, ncls = 0;  // patch: window rows h_0
    int patch_x = 0;                             // window columns w_0
    std::vector<int> pool_k, pool_kx;            // pool strides (the radix of the fragment grid), rows, columns, in layer order
    int S = 1, Sx = 1, F = 1;                    // products of the pool strides per axis; fragments
    int device = 0;
    bool head_fc = false;     // last layer fused into the head
    size_t head_w_off = 0, head_b_off = 0;
    size_t head_wp_off = 0;   // head weights in the previous layer's (block, row) order
    size_t head_wbf_off = 0;  // ... as bf16 row operands (ConvArgs::head_wbf), bf16 nets with paired blocks
    bool has_head_wbf = false;
    int ncu = 0;              // compute units of the device (0: plan-only net)
    int head_cin = 0;
    void *d_mem = nullptr;
    size_t mem_bytes = 0;
    PlanCache *plans = nullptr;  // owned; shared by the scans of all threads (locked inside)
    ~fs_net();
};

namespace {

int kstep_of(int dtype) { return dtype == DT_BF16 ? 32 : 16; }
int elem_of(int dtype) { return dtype == DT_BF16 ? 2 : 4; }

// Pack OIHW weights for the conv kernel: for K step s, channel block nb and
// lane (g = lane / 16, n = lane % 16) the LPE consecutive elements
// e = 0..LPE-1 hold W[nb*16 + n][ci][dy][dx] for the K index
//   vector path: tap = s / (cin / KSTEP), ci = (s % (cin / KSTEP)) * KSTEP + g*LPE + e
//   gather path: kk = s*KSTEP + g*LPE + e, tap = kk / cin, ci = kk % cin
// with tap = dy * k + dx; zero where the channel or K index is past the end.
// Output channel computed by row `row` of channel block `blk`.  The products
// leave row 4g + e of a block in lane (pixel, g), element e, so a lane holds
// four rows of every block.  bfloat16 layers whose waves own an even number
// of blocks pair blocks (2p, 2p + 1): rows 4g .. 4g + 3 of the pair are
// channels 32p + 8g + 0..3 and 32p + 8g + 4..7, eight consecutive channels
// that leave in one 16-byte store; otherwise block rows are channels in order
// (four consecutive float32 channels are 16 bytes already).
int chan_of(const NetLayer &l, int dtype, int blk, int row)
{
    if (dtype != DT_BF16 || (l.nb % 2) != 0) return blk * 16 + row;
    const int p = blk / 2, h = blk % 2, g = row / 4, e = row % 4;
    return 32 * p + 8 * g + 4 * h + e;
}

void pack_conv_weights(const NetLayer &l, const float *w, int dtype, std::vector<uint8_t> &out)
{
    const int KSTEP = kstep_of(dtype), LPE = KSTEP / 4, es = elem_of(dtype);
    const size_t n = (size_t)l.ksteps * l.nbt * 64 * LPE;
    out.assign(n * es, 0);
    const int taps = l.k * l.kx;
    for (int s = 0; s < l.ksteps; ++s)
        for (int nb = 0; nb < l.nbt; ++nb)
            for (int lane = 0; lane < 64; ++lane)
                for (int e = 0; e < LPE; ++e) {
                    const int g = lane / 16, nn = lane % 16;
                    const int co = chan_of(l, dtype, nb, nn);
                    int tap, ci;
                    if (l.vec) {
                        const int ncc = l.cin / KSTEP;
                        tap = s / ncc;
                        ci = (s % ncc) * KSTEP + g * LPE + e;
                    } else {
                        const int kk = s * KSTEP + g * LPE + e;
                        tap = kk / l.cin;
                        ci = kk % l.cin;
                    }
                    float v = 0.f;
                    if (co < l.cout && tap < taps) {
                        const int dy = tap / l.kx, dx = tap % l.kx;
                        v = w[(((size_t)co * l.cin + ci) * l.k + dy) * l.kx + dx];
                    }
                    const size_t idx = (((size_t)s * l.nbt + nb) * 64 + lane) * LPE + e;
                    if (dtype == DT_BF16) {
                        const uint16_t h = host_f2bf(v);
                        std::memcpy(&out[idx * 2], &h, 2);
                    } else {
                        std::memcpy(&out[idx * 4], &v, 4);
                    }
                }
}

// Optional tile override for tuning sweeps:
// FRAGSCAN_TILE="L:MB,NB,WN[,BAND[,WK[,LDS]]];..." (L = layer index, LDS = least
// dynamic LDS bytes per workgroup, which caps the workgroups per CU); any
// field <= 0 keeps the planner's choice.
bool tile_override(int layer, int *mb, int *nb, int *wn, int *band, int *wk = nullptr, int *lds = nullptr)
{
    const char *env = getenv("FRAGSCAN_TILE");
    if (!env) return false;
    const char *p = env;
    while (*p) {
        int L = -1, a = 0, b = 0, c = 0, d = 0, e = 0, f = 0;
        const int n = sscanf(p, "%d:%d,%d,%d,%d,%d,%d", &L, &a, &b, &c, &d, &e, &f);
        if (n >= 4 && L == layer) {
            if (mb && a > 0) *mb = a;
            if (nb && b > 0) *nb = b;
            if (wn && c > 0) *wn = c;
            if (band && n >= 5 && d > 0) *band = d;
            if (wk && n >= 6 && e > 0) *wk = e;
            if (lds && n >= 7 && f > 0) *lds = f;
            return true;
        }
        const char *semi = strchr(p, ';');
        if (!semi) break;
        p = semi + 1;
    }
    return false;
}

// Output-channel split of a conv layer: nb blocks of 16 channels per wave and
// wn waves across the channels; the channel blocks are padded to nb * wn.
void choose_channel_tile(int nbt, bool vec, int *nb, int *wn)
{
    if (!vec || nbt <= 4) {
        *wn = 1;
        *nb = std::min(nbt, 4);
        if (*nb == 0) *nb = 1;
        return;
    }
    if (nbt == 7) {  // one wave owns all seven blocks (no padding block)
        *wn = 1;
        *nb = 7;
        return;
    }
    *wn = 2;
    *nb = nbt <= 8 ? 4 : 7;
}

// ---------------------------------------------------------------------------
// Per-scan plan
// ---------------------------------------------------------------------------

struct Geo {  // fragment set entering a layer
    int Qy = 1, Qx = 1;           // fragments per axis; F = Qy * Qx per image
    std::vector<int> ey, ex;      // true sizes per y / x index
    int hmax = 0, wmax = 0, C = 0;
    bool is_image = true;         // the input image (float32 even in bf16 nets)
};

struct Launch {
    int type;                 // 0 conv, 1 pool, 2 head
    int layer, n_layers;
    int src, dst;             // -1 image, 0/1 workspace buffers, 2 output
    bool in_f32;
    ConvArgs conv;
    PoolArgs pool;
    HeadArgs head;
    int mb = 0, nb = 0, wn = 1, wk = 1;
    bool vec = false, has_fc = false;
    bool direct = false;      // vector-ALU convolution for tiny K
    int frag_tiles = 0, frag_lds = 0;  // per-fragment tiling when run tiles are planned
    int gx = 1, gy = 1;
    int frags = 0;
    long long out_pixels = 0;
    double flops = 0, bytes = 0;
    std::string name;
};

// A scan of a sub-image: the image region read has the image's pitch (rows
// per image img_h, pixels per row img_w) and starts img_off floats in; the
// outputs go into a map of out_h x out_w windows per image, out_off floats in.
struct View {
    int img_h = 0, img_w = 0;
    size_t img_off = 0;
    int out_h = 0, out_w = 0;
    size_t out_off = 0;
};

struct Plan {
    int B, H, W, ny, nx;
    View view;                 // img_h == 0: the whole image, outputs dense
    std::vector<Launch> launches;
    size_t buf_bytes = 0;      // each of the two ping-pong buffers
    size_t ws_bytes = 0;
    double flops = 0, bytes = 0;
};

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Workgroups of one launch dimension: HIP takes fewer than 2^32 work-items
// per dimension (256 per workgroup here).
constexpr long long kMaxGrid = (1LL << 32) / 256;

void fill_axis(AxisTable &t, const Geo &g)
{
    std::memset(&t, 0, sizeof t);
    for (int i = 0; i < g.Qy; ++i) t.y[i] = (uint16_t)g.ey[i];
    for (int i = 0; i < g.Qx; ++i) t.x[i] = (uint16_t)g.ex[i];
}

long long true_pixels(const Geo &g)
{
    long long sy = 0, sx = 0;
    for (int v : g.ey) sy += v;
    for (int v : g.ex) sx += v;
    return sy * sx;  // separable: sum over (fy, fx) of ey[fy] * ex[fx]
}

// Run tiles for a one-band layer: mt consecutive output pixels of the
// image's fragment sequence per tile instead of per fragment, whose tiles
// are counted for the largest fragment and leave the smaller ones' last
// tiles part empty (N4's 3x3 layer on a 448 x 448 image: 22-23 outputs per
// axis, 5 tiles of 128 per fragment where 4 hold the 22 x 22 ones).  A tile
// then spans at most two fragments, which needs every fragment to hold at
// least mt outputs; its window stacks the rows of both.  Planned when the
// LDS still fits and FRAGSCAN_RUN is not 0; make_plan then keeps them where
// they save a round of workgroups.
void plan_run_tiles(const NetLayer &l, const Geo &in, int mt, int cs, int es, int offtab, size_t other,
                    Launch &L)
{
    if (const char *e = getenv("FRAGSCAN_RUN"); e && e[0] == '0') return;
    if (!conv_tile_supported(L.mb, l.nb, l.wn, l.wk, l.vec, true)) return;
    const int ky = l.k, kx = l.kx;
    if (in.Qy > kMaxAxis || in.Qx > kMaxAxis) return;
    long long sy = 0, sx = 0;
    int hmin = 1 << 30, wmin = 1 << 30, wmax = 0;
    ConvArgs &a = L.conv;
    a.run_ypre[0] = a.run_xpre[0] = 0;
    for (int i = 0; i < in.Qy; ++i) {
        const int ho = in.ey[i] - ky + 1;
        hmin = std::min(hmin, ho);
        sy += std::max(ho, 0);
        if (sy >= 65536) return;  // uint16 prefix sums
        a.run_ypre[i + 1] = (uint16_t)sy;
    }
    for (int i = 0; i < in.Qx; ++i) {
        const int wo = in.ex[i] - kx + 1;
        wmin = std::min(wmin, wo);
        wmax = std::max(wmax, wo);
        sx += std::max(wo, 0);
        if (sx >= 65536) return;
        a.run_xpre[i + 1] = (uint16_t)sx;
    }
    if (hmin <= 0 || wmin <= 0 || (long long)hmin * wmin < mt || sy * sx >= (1LL << 31)) return;
    // window rows of a tile: n0 pixels of one fragment from any column span
    // at most (n0 + w - 2) / w + 1 output rows, the n1 = mt - n0 of the next
    // (from its column 0) (n1 - 1) / w + 1, each plus k_y - 1
    const int rows = (mt + wmin - 1) / wmin + 2 * ky;
    const size_t lds = offtab + (size_t)rows * (wmax + kx - 1) * cs * es;
    const size_t need = std::max(std::max(lds, other), (size_t)a.lds_bytes);
    if (need > kMaxLdsBytes) return;
    L.frag_tiles = a.tiles_per_band;
    L.frag_lds = a.lds_bytes;
    a.run = 1;
    a.run_pix = (int)(sy * sx);
    a.run_wsum = (int)sx;
    a.tiles_per_band = (int)((sy * sx + mt - 1) / mt);
    a.lds_bytes = (int)need;
}

// Tile choice for a conv launch (the tiling itself is described in conv_impl.h).
// wide: the float32 4 x 13 tile of conv_f32_wide.hip (l.nb = 13, l.wn = 1),
// which has no entry in the shared tile lists.
fs_status plan_conv_tiles(const fs_net *net, const NetLayer &l, const Geo &in, Launch &L, bool wide = false)
{
    const int ky = l.k, kx = l.kx;
    const int hout_max = in.hmax - ky + 1, wout_max = in.wmax - kx + 1;
    const int es = elem_of(net->dtype);
    const int KSTEP = kstep_of(net->dtype);
    // pixel stride in LDS: +16 bytes per pixel spreads 16 consecutive pixels'
    // 16-byte reads over distinct banks (FRAGSCAN_LDS_PAD overrides, elements)
    int pad = 16 / es;
    if (const char *e = getenv("FRAGSCAN_LDS_PAD")) pad = atoi(e);
    if (l.vec && (pad * es) % 16) pad = 16 / es;
    const int cs = l.vec ? l.cin + pad : l.cin;
    const int offtab = l.vec ? 0 : (int)align_up((size_t)l.ksteps * KSTEP * 4, 16);
    // distinct output widths present; every fragment's output height and width
    std::vector<int> wouts, houts, wouts_all;
    for (int v : in.ex)
        if (v - kx + 1 > 0 && std::find(wouts.begin(), wouts.end(), v - kx + 1) == wouts.end())
            wouts.push_back(v - kx + 1);
    for (int v : in.ey)
        if (v - ky + 1 > 0) houts.push_back(v - ky + 1);
    for (int v : in.ex)
        if (v - kx + 1 > 0) wouts_all.push_back(v - kx + 1);
    const int wm = 4 / (l.wn * l.wk);
    int mb_force = 0, band_force = 0, lds_min = 0;
    tile_override(L.layer, &mb_force, nullptr, nullptr, &band_force, nullptr, &lds_min);
    // pixel blocks per wave: four (more products per operand load; measured
    // faster on every conv layer of the five workloads, including the short
    // K walks of workload 3's 2x2x16 -> 100 layer, 742 -> 688 us against two,
    // and workload 5's gathered 3x3x3 -> 32 first layer), else the neighbours
    const int mbs[4] = {4, 2, 1, 8};
    for (int mi = 0; mi < 4; ++mi) {
        const int mb = mb_force ? mb_force : mbs[mi];
        if (wide ? mb != 4 : !conv_tile_supported(mb, l.nb, l.wn, l.wk, l.vec)) {
            if (mb_force) break;
            continue;
        }
        const int mt = 16 * mb * wm;
        // bands of about 16 columns keep the window (and LDS) small enough
        // for several workgroups per CU
        int nbands = wout_max <= 32 ? 1 : (wout_max + 15) / 16;
        if (band_force) nbands = (wout_max + band_force - 1) / band_force;
        for (; nbands <= wout_max; ++nbands) {
            const int band_w = (wout_max + nbands - 1) / nbands;
            // the kernel's index arithmetic (Div in conv_impl.h) takes pixel
            // numbers within a band below 2^20
            if ((long long)hout_max * band_w >= (1 << 20)) continue;
            const size_t red = (size_t)l.wn * mt * kMaxFusedClasses * 4;  // fused-head reduction
            // split-K partial sums of the waves with wk > 0
            const size_t part = (size_t)(l.wk - 1) * (4 / l.wk) * mb * l.nb * 4 * 64 * 4;
            // Stores: straight from the registers (16-byte runs of 4 f32 or
            // 8 bf16 channels per lane; measured no slower than restaging on
            // every conv layer of the five workloads, faster on the bf16 and
            // 16-channel ones); FRAGSCAN_STORE=lds restages through an LDS
            // tile [mt][wn*nb*16 + 16 bytes] and writes whole rows instead.
            int direct = 1;
            if (const char *e = getenv("FRAGSCAN_STORE"); e && e[0]) direct = e[0] == 'd';
            const size_t otile = direct ? 0 : (size_t)mt * (l.wn * l.nb * 16 + 16 / es) * es;
            const size_t other = std::max(std::max(part, red), std::max(otile, (size_t)lds_min));
            // Pixel tiles: mt consecutive pixels of a band, whose window in
            // the narrowest band spans the most rows, and that sizes the LDS
            // of every workgroup.  Row tiles (several bands): rows_t = mt /
            // band_w whole band rows, the same window rows in every band.
            // (the window of a tile in a band of width t spans the rows its
            // pixels touch plus k_y - 1, and t + k_x - 1 columns: the largest over
            // the bands present and the tile starts i * mt, which repeat
            // with period t)
            size_t lds_p = 0;
            for (int wo : wouts)
                for (int b = 0; b < nbands; ++b) {
                    const int t = std::min(band_w, wo - b * band_w);
                    if (t <= 0) break;
                    int span = 0;
                    for (int i = 0; i < t; ++i) span = std::max(span, (int)(((long long)i * mt) % t + mt - 1) / t + 1);
                    const int rows = std::min(span + ky - 1, in.hmax);
                    lds_p = std::max(lds_p, offtab + (size_t)rows * (t + kx - 1) * cs * es);
                }
            const int rows_t = (nbands > 1 && mt >= band_w) ? mt / band_w : 0;
            const size_t lds_r = rows_t ? offtab + (size_t)std::min(rows_t + ky - 1, in.hmax) * (band_w + kx - 1) * cs * es
                                        : lds_p;
            if (std::min(lds_p, lds_r) > 96 * 1024) {
                if (band_w <= 8) break;
                continue;
            }
            const size_t need_p = std::max(lds_p, other), need_r = std::max(lds_r, other);
            // Which one: the tiles that hold pixels, weighted by how much a
            // lone workgroup per CU (nothing to overlap its staging and
            // epilogue with) or two cost against three or more; measured on
            // N4's 48 -> 48 layers: 1 -> 2 per CU 15% faster (5x5 on 606^2
            // images), 2 -> 3 at most 4% and outweighed by the row tiles'
            // extra part-empty tiles.  FRAGSCAN_ROWTILES=1/0 forces either.
            bool use_rows = false;
            if (rows_t && need_r <= kMaxLdsBytes) {
                auto per_cu = [&](size_t need) {
                    if (net->ncu > 0)
                        return conv_blocks_per_cu(net->dtype, in.is_image, mb, l.nb, l.wn, l.wk, l.vec, false,
                                                  (int)need);
                    return (int)std::min<size_t>(8, kMaxLdsBytes / need);
                };
                auto weight = [](int n) { return n <= 1 ? 1.30 : n == 2 ? 1.02 : 1.0; };
                long long tiles_p = 0, tiles_r = 0;
                for (int ho : houts)
                    for (int wo : wouts_all)
                        for (int b = 0; b < nbands; ++b) {
                            const int twb = std::min(band_w, wo - b * band_w);
                            if (twb <= 0) break;
                            tiles_p += ((long long)ho * twb + mt - 1) / mt;
                            tiles_r += (ho + rows_t - 1) / rows_t;
                        }
                const double cost_p = need_p <= kMaxLdsBytes ? tiles_p * weight(per_cu(need_p)) : 1e300;
                const double cost_r = tiles_r * weight(per_cu(need_r));
                use_rows = cost_r < cost_p;
                if (const char *e = getenv("FRAGSCAN_ROWTILES"); e && e[0]) use_rows = e[0] == '1';
            }
            const size_t need = use_rows ? need_r : need_p;
            if (need > kMaxLdsBytes) {
                if (mb_force) break;
                continue;
            }
            L.mb = mb;
            L.conv.band_w = band_w;
            L.conv.nbands = nbands;
            L.conv.mt = mt;
            L.conv.tile_rows = use_rows ? rows_t : 0;
            L.conv.tiles_per_band = use_rows ? (hout_max + rows_t - 1) / rows_t : (hout_max * band_w + mt - 1) / mt;
            L.conv.lds_cs = cs;
            L.conv.direct_store = direct;
            L.conv.lds_bytes = (int)need;
            L.conv.run = 0;
            if (nbands == 1 && direct) plan_run_tiles(l, in, mt, cs, es, offtab, std::max(part, red), L);
            return FS_OK;
        }
        if (mb_force) break;
    }
    return fail(FS_ERR_UNSUPPORTED, "layer %d: no convolution tile fits in LDS", L.layer);
}

// Children of a ky x kx pool with strides sy x sx (Eqs. 5-7, per axis; the
// paper's pools have s = k): parent index i and offset o < s give child
// i*s + o, holding the windows o, o + s, ... that end inside the parent:
// floor((n - o - k + s) / s) of them for a parent of size n, never below 0.
Geo pool_geo(const Geo &g, int ky, int kx, int sy, int sx)
{
    Geo o;
    o.Qy = g.Qy * sy;
    o.Qx = g.Qx * sx;
    o.ey.assign(o.Qy, 0);
    o.ex.assign(o.Qx, 0);
    for (int i = 0; i < g.Qy; ++i)
        for (int off = 0; off < sy; ++off) o.ey[i * sy + off] = std::max(g.ey[i] - off - ky + sy, 0) / sy;
    for (int i = 0; i < g.Qx; ++i)
        for (int off = 0; off < sx; ++off) o.ex[i * sx + off] = std::max(g.ex[i] - off - kx + sx, 0) / sx;
    o.C = g.C;
    o.hmax = *std::max_element(o.ey.begin(), o.ey.end());
    o.wmax = *std::max_element(o.ex.begin(), o.ex.end());
    o.is_image = false;
    return o;
}

// Tiles of a convolution with the following kpy x kpx pool fused in (kernel:
// conv_impl.h, pool_ky > 0).  Bands of ~16 columns of the stride-1 max
// filter; a tile holds pool_rt filter rows, i.e. (pool_rt + kpy - 1) x
// (band + kpx - 1) convolution outputs, which must fit the register tile (mt
// pixels).
fs_status plan_conv_pool_tiles(const fs_net *net, const NetLayer &l, const Geo &in, int kpy, int kpx, Launch &L)
{
    const int ky = l.k, kx = l.kx;
    const int es = elem_of(net->dtype);
    const int KSTEP = kstep_of(net->dtype);
    const int pad = 16 / es;
    const int cs = l.vec ? l.cin + pad : l.cin;
    const int offtab = l.vec ? 0 : (int)align_up((size_t)l.ksteps * KSTEP * 4, 16);
    const int hM_max = in.hmax - ky + 1 - kpy + 1, wM_max = in.wmax - kx + 1 - kpx + 1;
    const int wm = 4 / (l.wn * l.wk);
    int mb_force = 0, band_force = 0;
    tile_override(L.layer, &mb_force, nullptr, nullptr, &band_force);
    const int mbs[4] = {4, 8, 2, 1};
    for (int mi = 0; mi < 4; ++mi) {
        const int mb = mb_force ? mb_force : mbs[mi];
        if (!conv_tile_supported(mb, l.nb, l.wn, l.wk, l.vec)) {
            if (mb_force) break;
            continue;
        }
        const int mt = 16 * mb * wm;
        const int wmax = std::max(wM_max, 1), hmax = std::max(hM_max, 1);
        int nbands = wmax <= 32 ? 1 : (wmax + 15) / 16;
        if (band_force) nbands = (wmax + band_force - 1) / band_force;
        for (; nbands <= wmax; ++nbands) {
            const int band_w = (wmax + nbands - 1) / nbands;
            const int ew = band_w + kpx - 1;
            const int rt = std::min(mt / ew - (kpy - 1), hmax);
            if (rt < 1) continue;  // narrower bands
            const size_t win = offtab + (size_t)(rt + kpy - 1 + ky - 1) * (ew + kx - 1) * cs * es;
            const size_t tile = (size_t)mt * (l.wn * l.nb * 16 + pad) * es;
            const size_t part = (size_t)(l.wk - 1) * (4 / l.wk) * mb * l.nb * 4 * 64 * 4;
            const size_t need = std::max(std::max(win, tile), part);
            if (win > 96 * 1024 || need > kMaxLdsBytes) {
                if (band_w <= 8) break;
                continue;
            }
            if ((long long)in.hmax * ew >= (1 << 20)) continue;
            L.mb = mb;
            L.conv.band_w = band_w;
            L.conv.nbands = nbands;
            L.conv.mt = mt;
            L.conv.pool_rt = rt;
            L.conv.tiles_per_band = (hmax + rt - 1) / rt;
            L.conv.lds_cs = cs;
            L.conv.direct_store = 1;
            L.conv.lds_bytes = (int)need;
            return FS_OK;
        }
        if (mb_force) break;
    }
    return fail(FS_ERR_UNSUPPORTED, "layer %d: no fused convolution + pool tile", L.layer);
}

// Whether the pool after conv layer li goes into the convolution's epilogue.
// Per output pixel, fusing recomputes a halo share `ov` of the products
// (2 c_in k^2 c_out ov FLOPs; ov ~ 0.35 for 2 x 2 pools with 16-column
// bands, 0.5 for larger pools) and saves the pool's read and write of the
// pixel (2 c_out elem bytes).  At peak rates that pays when
// c_in k^2 ov < elem * (peak FLOP/s / HBM bytes/s): every layer of the five
// workloads except N4's 48 -> 48 convolutions, whose fused form measured
// 10-35% slower.  FRAGSCAN_POOL_FUSE=1 / 0 forces it on / off.
bool want_pool_fusion(const fs_net *net, int li)
{
    const int nl = (int)net->L.size();
    if (li + 1 >= nl) return false;
    const NetLayer &l = net->L[li], &p = net->L[li + 1];
    if (l.kind == FS_MAXPOOL || p.kind != FS_MAXPOOL || l.nbt != l.nb * l.wn) return false;
    if (p.sy != p.k || p.sx != p.kx) return false;  // the fused walk samples the filter at steps of k
    if (const char *e = getenv("FRAGSCAN_POOL_FUSE"); e && e[0]) return e[0] == '1';
    const double ov = (p.k == 2 && p.kx == 2) ? 0.35 : 0.5;
    const double ridge = net->dtype == DT_BF16 ? 2516.6e12 / 8e12 : 157.3e12 / 8e12;  // FLOP per byte
    return (double)l.cin * l.k * l.kx * ov < elem_of(net->dtype) * ridge;
}

// First output coordinate (along one axis) of the final fragments' axis
// index f: its offsets at the successive pools, sizes ks (first pool first),
// are the mixed-radix digits of f read most significant first, and the
// window offset they select is sum o_m * (k_1 * ... * k_{m-1}).
int axis_base(const std::vector<int> &ks, int S, int f)
{
    int rest = f, base = 0;
    for (int m = (int)ks.size() - 1; m >= 0; --m) {
        S /= ks[m];
        base += (rest % ks[m]) * S;
        rest /= ks[m];
    }
    return base;
}

fs_status make_plan(const fs_net *net, int B, int H, int W, Plan &P, const View *view = nullptr)
{
    if (B < 1 || H < 1 || W < 1) return fail(FS_ERR_SHAPE, "B, H, W must be >= 1");
    if (H < net->patch || W < net->patch_x)
        return fail(FS_ERR_SHAPE, "image %dx%d smaller than the window %dx%d", H, W, net->patch, net->patch_x);
    // fragment sizes travel as 16-bit per-axis tables; a larger image (or
    // tiled-scan region) goes through fs_scan_tiled with fewer rows / columns
    if (H > kMaxSide || W > kMaxSide)
        return fail(FS_ERR_UNSUPPORTED, "image (or tile region) %dx%d has a side above %d; scan it in tiles "
                    "(fs_scan_tiled) of fewer rows / columns", H, W, kMaxSide);
    // fragment batch indices (B * F) and per-launch fragment counts are int
    if ((long long)B * net->F >= (1LL << 24))
        return fail(FS_ERR_UNSUPPORTED, "batch %d x %d fragments: scan fewer images per call", B, net->F);
    P = Plan();
    P.B = B;
    P.H = H;
    P.W = W;
    P.ny = H - net->patch + 1;
    P.nx = W - net->patch_x + 1;
    if (view) P.view = *view;
    // the image's pitch (a view reads a region of a larger image) and the
    // output map's (a view writes a region of a larger map)
    const int img_h = view ? view->img_h : H, img_w = view ? view->img_w : W;
    const int map_h = view ? view->out_h : P.ny, map_w = view ? view->out_w : P.nx;
    const int es = elem_of(net->dtype);

    Geo g;
    g.Qy = g.Qx = 1;
    g.ey = {H};
    g.ex = {W};
    g.hmax = H;
    g.wmax = W;
    g.C = net->C;
    g.is_image = true;

    const int nl = (int)net->L.size();
    const int body = net->head_fc ? nl - 1 : nl;
    // the last 1x1 layer goes into the epilogue of the layer before it when
    // that is a convolution whose workgroups cover all its channels
    bool fuse = false;
    if (net->head_fc && net->ncls <= kMaxFusedClasses && nl >= 2) {
        const NetLayer &pl = net->L[nl - 2];
        fuse = pl.kind != FS_MAXPOOL && pl.nbt == pl.nb * pl.wn && !getenv("FRAGSCAN_NO_FUSED_HEAD");
    }
    int cur = -1;  // where the current activations live
    size_t buf = 0;
    for (int li = 0; li < body; ++li) {
        const NetLayer &l = net->L[li];
        Launch L{};
        L.layer = li;
        L.n_layers = 1;
        L.src = cur;
        L.dst = (cur == 0) ? 1 : 0;
        L.in_f32 = g.is_image;
        const int F = g.Qy * g.Qx;
        const long long in_pix = true_pixels(g);
        Geo o;
        if (l.kind == 1) {  // pool
            const int ky = l.k, kx = l.kx;
            if (g.Qy * l.sy > kMaxAxis || g.Qx * l.sx > kMaxAxis)
                return fail(FS_ERR_UNSUPPORTED, "more than %d fragments per axis", kMaxAxis);
            o = pool_geo(g, ky, kx, l.sy, l.sx);
            L.type = 1;
            if (g.is_image && view) return fail(FS_ERR_UNSUPPORTED, "a tiled scan needs a convolution first");
            PoolArgs &a = L.pool;
            a.F = F;
            a.Qx = g.Qx;
            a.in_h = g.hmax;
            a.in_w = g.wmax;
            a.out_h = std::max(o.hmax, 1);
            a.out_w = std::max(o.wmax, 1);
            a.C = g.C;
            a.ky = ky;
            a.kx = kx;
            a.sy = l.sy;
            a.sx = l.sx;
            a.n_children = B * F * l.sy * l.sx;
            // Row-band kernel: 8 filter rows per thread, or 4 where that
            // still leaves at least 32 workgroups per CU (more threads in
            // flight: N4's pools on 8 x 1024^2 images 2-5% faster; on one
            // 512^2 image, 2-5% slower).  FRAGSCAN_POOL_ROWS=4/8 forces it.
            {
                const int vpp = (net->dtype == DT_F32 && g.C % 4 == 0) ? g.C / 4
                                : (net->dtype == DT_BF16 && !g.is_image && g.C % 8 == 0) ? g.C / 8 : g.C;
                const long long wg8 = (long long)B * F * ((g.hmax + 7) / 8) * (((long long)g.wmax * vpp + 255) / 256);
                a.rows = wg8 >= 32LL * (net->ncu > 0 ? net->ncu : 256) ? 4 : 8;
                if (const char *e = getenv("FRAGSCAN_POOL_ROWS")) a.rows = atoi(e) == 4 ? 4 : 8;
            }
            fill_axis(a.ext, g);
            L.gx = (int)std::min<long long>((long long)B * F * l.sy * l.sx * a.out_h, kMaxGrid);
            L.frags = B * F * l.sy * l.sx;
            L.out_pixels = (long long)B * true_pixels(o);
            L.bytes = (double)B * in_pix * g.C * (g.is_image ? 4 : es) + (double)L.out_pixels * o.C * es;
            L.name = pool_kernel_name(net->dtype, g.is_image, ky, kx, l.sy, l.sx, g.C, a.rows);
        } else {  // conv or fc as convolution
            const int ky = l.k, kx = l.kx;
            o.Qy = g.Qy;
            o.Qx = g.Qx;
            o.ey.resize(g.Qy);
            o.ex.resize(g.Qx);
            for (int i = 0; i < g.Qy; ++i) o.ey[i] = std::max(g.ey[i] - (ky - 1), 0);
            for (int i = 0; i < g.Qx; ++i) o.ex[i] = std::max(g.ex[i] - (kx - 1), 0);
            o.C = l.cout;
            o.hmax = *std::max_element(o.ey.begin(), o.ey.end());
            o.wmax = *std::max_element(o.ex.begin(), o.ex.end());
            L.type = 0;
            L.vec = l.vec;
            L.nb = l.nb;
            L.wn = l.wn;
            L.wk = l.wk;
            ConvArgs &a = L.conv;
            a.nfrag = B * F;
            a.F = F;
            a.Qy = g.Qy;
            a.Qx = g.Qx;
            a.in_h = g.is_image ? img_h : g.hmax;  // fragment stride and row pitch
            a.in_w = g.is_image ? img_w : g.wmax;
            a.in_c = g.C;
            a.out_h = std::max(o.hmax, 1);
            a.out_w = std::max(o.wmax, 1);
            a.ky = ky;
            a.kx = kx;
            a.cin = l.cin;
            a.cout = l.cout;
            // the last layer, when not fused into the head, leaves its
            // activation to the head (softmax needs all classes)
            a.act = (li == nl - 1) ? ACT_NONE : l.act;
            a.ksteps = l.ksteps;
            a.nbt = l.nbt;
            a.nbu = (l.cout + 15) / 16;
            fill_axis(a.ext, g);
            const bool fused_here = fuse && li == body - 1;
            // Small-K layers with one 16-channel output block reuse each
            // gathered A fragment only once on the matrix cores; there the
            // per-pixel vector-ALU kernel is faster.  FRAGSCAN_DIRECT=1 takes
            // it for every layer it supports, =0 for none.
            const char *dv = getenv("FRAGSCAN_DIRECT");
            const bool want_direct = dv ? dv[0] == '1' : l.cout <= 16;
            const bool pool_fuse = !fused_here && want_pool_fusion(net, li);
            if (l.has_w32 && !fused_here && !pool_fuse && want_direct) {
                L.direct = true;
                L.conv.lds_bytes = 0;
            } else {
                fs_status st = pool_fuse ? plan_conv_pool_tiles(net, l, g, net->L[li + 1].k, net->L[li + 1].kx, L)
                                         : plan_conv_tiles(net, l, g, L);
                if (st != FS_OK) return st;
                // The float32 FC layer with the fused head on a grid that
                // runs it one workgroup per CU (the rule below), with 14
                // blocks of 16 for at most 208 channels (200 in N4): the
                // 4 x 13 tile drops the padding block and covers 256 pixels
                // per workgroup (N4 on 512 x 512: 305 -> 286 us; on larger
                // grids, where the 7 x 2 tiles run two per CU, 14% slower).
                // FRAGSCAN_WIDE=1 / 0 forces it on / off where it applies.
                if (fused_here && !pool_fuse && net->dtype == DT_F32 && l.vec && l.nb == 7 && l.wn == 2 &&
                    l.wk == 1 && l.nbt == 14 && l.cout <= 13 * 16) {
                    const long long tiles = (long long)B * F * a.nbands * (a.run ? L.frag_tiles : a.tiles_per_band);
                    bool wide = net->ncu > 0 && tiles <= 12LL * net->ncu &&
                                conv_blocks_per_cu(net->dtype, g.is_image, L.mb, l.nb, l.wn, l.wk, l.vec, false,
                                                   a.lds_bytes) == 2;
                    if (const char *e = getenv("FRAGSCAN_WIDE"); e && e[0]) wide = e[0] == '1';
                    if (wide) {
                        NetLayer lw = l;
                        lw.nb = 13;
                        lw.wn = 1;
                        Launch Lw = L;
                        Lw.nb = 13;
                        Lw.wn = 1;
                        Lw.conv.run = 0;
                        if (plan_conv_tiles(net, lw, g, Lw, true) == FS_OK) L = Lw;
                    }
                }
            }
            L.gy = L.direct ? 1 : std::max(l.nbt / (L.nb * L.wn), 1);
            if (L.direct) {
                L.gx = (int)std::min<long long>((long long)B * F * (((long long)a.out_h * a.out_w + 255) / 256),
                                                kMaxGrid);
            } else {
                // grid (a multiple of 8 for the XCD-contiguous tile order)
                // and dynamic LDS of either tiling; returns the rounds of
                // workgroups the device needs for it
                auto finish = [&](bool run, long long tiles, int &lds, int &gx) {
                    gx = (int)std::min<long long>((tiles + 7) / 8 * 8, kMaxGrid);
                    // The FC layer with the fused head, when its register
                    // tile fits only two workgroups per CU, ran 2-7% faster
                    // one per CU on grids of at most 12 workgroups per CU
                    // (N4 on 512x512 and 2x512x512 images; 3-5% slower on
                    // larger grids; other layers, whose tiles fit three,
                    // 12-18% slower): pad its LDS to admit one.
                    if (fused_here && net->ncu > 0 && (long long)gx * L.gy <= 12LL * net->ncu &&
                        conv_blocks_per_cu(net->dtype, g.is_image, L.mb, L.nb, L.wn, L.wk, L.vec, run, lds) == 2)
                        lds = std::max(lds, (int)(kMaxLdsBytes / 2 + 1024));
                    // plan-only nets: 256 CUs, one workgroup each
                    const int bpc = net->ncu > 0 ? conv_blocks_per_cu(net->dtype, g.is_image, L.mb, L.nb, L.wn,
                                                                      L.wk, L.vec, run, lds) : 1;
                    const long long slots = (long long)(net->ncu > 0 ? net->ncu : 256) * std::max(bpc, 1);
                    return ((long long)gx * L.gy + slots - 1) / slots;
                };
                int lds = a.lds_bytes, gx = 0;
                const long long rounds =
                    finish(a.run, (long long)(a.run ? B : B * F) * a.nbands * a.tiles_per_band, lds, gx);
                if (a.run) {
                    // Run tiles only where they save a round of workgroups:
                    // with equal rounds their two-fragment windows cost
                    // 2% (N4's 3x3 layer on 512 x 512: 1375 run tiles
                    // against 1536, 6 rounds each); FRAGSCAN_RUN=1 keeps them.
                    int lds_f = L.frag_lds, gx_f = 0;
                    const long long rounds_f = finish(false, (long long)B * F * L.frag_tiles, lds_f, gx_f);
                    const char *e = getenv("FRAGSCAN_RUN");
                    if (rounds >= rounds_f && !(e && e[0] == '1')) {
                        a.run = 0;
                        a.tiles_per_band = L.frag_tiles;
                        lds = lds_f;
                        gx = gx_f;
                    }
                }
                a.lds_bytes = lds;
                L.gx = gx;
            }
            L.frags = B * F;
            L.out_pixels = (long long)B * true_pixels(o);
            L.flops = (double)L.out_pixels * 2.0 * l.cin * ky * kx * l.cout;
            L.bytes = (double)B * in_pix * g.C * (g.is_image ? 4 : es) + (double)L.out_pixels * l.cout * es +
                      (double)l.cin * ky * kx * l.cout * es;
            L.name = L.direct ? conv_direct_kernel_name(net->dtype, g.is_image, l.cin, ky * kx)
                              : conv_kernel_name(net->dtype, g.is_image, L.mb, L.nb, L.wn, L.wk, L.vec, a.run);
            if (pool_fuse) {
                const int kpy = net->L[li + 1].k, kpx = net->L[li + 1].kx;
                if (g.Qy * kpy > kMaxAxis || g.Qx * kpx > kMaxAxis)
                    return fail(FS_ERR_UNSUPPORTED, "more than %d fragments per axis", kMaxAxis);
                const Geo o2 = pool_geo(o, kpy, kpx, kpy, kpx);
                a.pool_ky = kpy;
                a.pool_kx = kpx;
                a.pool_oh = std::max(o2.hmax, 1);
                a.pool_ow = std::max(o2.wmax, 1);
                L.n_layers = 2;
                L.bytes = (double)B * in_pix * g.C * (g.is_image ? 4 : es) +
                          (double)B * true_pixels(o2) * l.cout * es + (double)l.cin * ky * kx * l.cout * es;
                L.name += "+pool";
                o = o2;
                ++li;  // the pool is done
            }
            if (fuse && li == body - 1) {
                const NetLayer &hl = net->L[nl - 1];
                if (net->dtype == DT_BF16 && L.nb % 2 == 0 && !net->has_head_wbf)
                    return fail(FS_ERR_UNSUPPORTED, "layer %d: no bf16 head operands for the fused head", li);
                a.head_ncls = net->ncls;
                a.head_act = hl.act;
                a.ny = map_h;  // output pitch
                a.nx = map_w;
                a.Sy = net->S;
                a.Sx = net->Sx;
                for (int f = 0; f < o.Qy; ++f) a.base_y[f] = (uint16_t)axis_base(net->pool_k, net->S, f);
                for (int f = 0; f < o.Qx; ++f) a.base_x[f] = (uint16_t)axis_base(net->pool_kx, net->Sx, f);
                // Fragment tiles in x-sibling order (ConvArgs::xsib):
                // FRAGSCAN_XSIB=0 keeps fragment order.
                const char *xs = getenv("FRAGSCAN_XSIB");
                a.xsib = !a.run && !(xs && xs[0] == '0');
                // Channel halves swapped in alternate workgroups where the
                // second half ends in padding (ConvArgs::swapn);
                // FRAGSCAN_SWAP=0 keeps them in place.
                const char *sw = getenv("FRAGSCAN_SWAP");
                a.swapn = a.nbu < a.nbt && !(sw && sw[0] == '0');
                L.dst = 2;
                L.n_layers = 2;
                const long long npix = (long long)B * P.ny * P.nx;
                L.flops += (double)npix * 2.0 * hl.cin * hl.cout;
                L.bytes = (double)B * in_pix * g.C * (g.is_image ? 4 : es) + (double)npix * net->ncls * 4 +
                          (double)l.cin * ky * kx * l.cout * es;
                L.name += "+head";
            }
            if (!L.direct && a.run) L.name += "+run";
        }
        o.is_image = false;
        // kernels address within one fragment (or image) with 32-bit offsets;
        // a tiled scan's first layer reads its region with the image's pitch
        if ((long long)std::max(o.hmax, 1) * std::max(o.wmax, 1) * o.C >= (1LL << 31) ||
            (long long)std::max(g.hmax, 1) * std::max(g.wmax, 1) * g.C >= (1LL << 31) ||
            (g.is_image && (long long)g.hmax * img_w * g.C >= (1LL << 31)))
            return fail(FS_ERR_UNSUPPORTED, "layer %d: a fragment holds 2^31 or more elements", li);
        if (L.gx >= kMaxGrid || L.gx < 1)
            return fail(FS_ERR_UNSUPPORTED, "layer %d: grid too large; scan the image in tiles", li);
        if (L.dst != 2) {
            const size_t out_bytes = (size_t)B * o.Qy * o.Qx * std::max(o.hmax, 1) * std::max(o.wmax, 1) * o.C * es;
            buf = std::max(buf, out_bytes);
        }
        P.flops += L.flops;
        P.bytes += L.bytes;
        P.launches.push_back(L);
        cur = L.dst;
        g = o;
    }

    // head: the (fused) last layer, its activation, and the reassembly
    if (!fuse) {
        Launch L{};
        L.type = 2;
        L.layer = net->head_fc ? nl - 1 : nl;
        L.n_layers = net->head_fc ? 1 : 0;
        L.src = cur;
        L.dst = 2;
        L.in_f32 = g.is_image;
        L.has_fc = net->head_fc;
        HeadArgs &a = L.head;
        a.B = B;
        a.F = g.Qy * g.Qx;
        a.Qx = g.Qx;
        a.in_h = std::max(g.hmax, 1);
        a.in_w = std::max(g.wmax, 1);
        if (g.is_image && view) return fail(FS_ERR_UNSUPPORTED, "a tiled scan needs a convolution first");
        a.C = g.C;
        a.ny = P.ny;
        a.nx = P.nx;
        a.out_ny = map_h;
        a.out_nx = map_w;
        a.ncls = net->ncls;
        a.act = net->L.back().act;
        a.Sy = net->S;
        a.Sx = net->Sx;
        // Y mod S -> per-axis fragment index: the mixed-radix digits of r
        // (least significant = first pool) read back most significant first
        auto digits = [](const std::vector<int> &ks, int S, uint16_t *map) {
            for (int r = 0; r < S; ++r) {
                int rr = r, idx = 0;
                for (int k : ks) {
                    idx = idx * k + rr % k;
                    rr /= k;
                }
                map[r] = (uint16_t)idx;
            }
        };
        digits(net->pool_k, net->S, a.digit_y);
        digits(net->pool_kx, net->Sx, a.digit_x);
        fill_axis(a.ext, g);
        const long long npix = (long long)B * P.ny * P.nx;
        // the head numbers a window within its image with 32-bit integers
        const long long per_wg = 256LL / kHeadLanesPerPixel * kHeadPixelsPerGroup;
        if ((long long)P.ny * P.nx >= (1LL << 31) || (npix + per_wg - 1) / per_wg >= kMaxGrid)
            return fail(FS_ERR_UNSUPPORTED, "%d x %d windows per image (batch %d): scan the image in tiles", P.ny,
                        P.nx, B);
        L.gx = (int)((npix + per_wg - 1) / per_wg);
        L.frags = B * a.F;
        L.out_pixels = npix;
        L.flops = net->head_fc ? (double)npix * 2.0 * net->head_cin * net->ncls : 0.0;
        L.bytes = (double)npix * g.C * (g.is_image ? 4 : es) + (double)npix * net->ncls * 4;
        L.name = head_kernel_name(net->dtype, g.is_image, net->head_fc);
        P.flops += L.flops;
        P.bytes += L.bytes;
        P.launches.push_back(L);
    }
    P.buf_bytes = align_up(buf, 256);
    P.ws_bytes = 2 * P.buf_bytes;
    return FS_OK;
}

}  // namespace

// Plans already made for a net, by batch, image size, view and the planner
// switches in the environment, so a scan repeated at the same size enqueues
// its launches without planning again.  Plans are immutable once made and
// shared through shared_ptr, so a plan stays valid for a scan that holds it
// while another thread adds plans.
struct PlanCache {
    struct Key {
        int B, H, W, img_h, img_w, out_h, out_w;
        std::string env;
        bool operator==(const Key &o) const
        {
            return B == o.B && H == o.H && W == o.W && img_h == o.img_h && img_w == o.img_w && out_h == o.out_h &&
                   out_w == o.out_w && env == o.env;
        }
    };
    static constexpr size_t kMax = 16;  // most recently used last
    std::mutex mu;
    std::vector<std::pair<Key, std::shared_ptr<const Plan>>> plans;
};

fs_net::~fs_net() { delete plans; }

namespace {

// The planner switches (tuning and test overrides) a plan was made under.
std::string planner_env()
{
    static const char *const vars[] = {"FRAGSCAN_TILE", "FRAGSCAN_DIRECT", "FRAGSCAN_POOL_FUSE",
                                       "FRAGSCAN_NO_FUSED_HEAD", "FRAGSCAN_RUN", "FRAGSCAN_ROWTILES",
                                       "FRAGSCAN_STORE", "FRAGSCAN_LDS_PAD", "FRAGSCAN_WIDE",
                                       "FRAGSCAN_POOL_ROWS", "FRAGSCAN_XSIB",
                                       "FRAGSCAN_SWAP"};
    std::string sig;
    for (const char *v : vars) {
        const char *e = getenv(v);
        sig += e ? e : "\x01";
        sig += '\x02';
    }
    return sig;
}

fs_status get_plan(const fs_net *net, int B, int H, int W, std::shared_ptr<const Plan> &out,
                   const View *view = nullptr)
{
    PlanCache::Key k{B, H, W, view ? view->img_h : 0, view ? view->img_w : 0, view ? view->out_h : 0,
                     view ? view->out_w : 0, planner_env()};
    PlanCache *c = net->plans;
    if (c) {
        std::lock_guard<std::mutex> lock(c->mu);
        for (size_t i = 0; i < c->plans.size(); ++i)
            if (c->plans[i].first == k) {
                out = c->plans[i].second;
                if (i + 1 != c->plans.size()) {  // move to the back (most recent)
                    auto e = c->plans[i];
                    c->plans.erase(c->plans.begin() + i);
                    c->plans.push_back(e);
                }
                return FS_OK;
            }
    }
    auto P = std::make_shared<Plan>();
    fs_status st = make_plan(net, B, H, W, *P, view);
    if (st != FS_OK) return st;
    out = P;
    if (c) {
        std::lock_guard<std::mutex> lock(c->mu);
        if (c->plans.size() >= PlanCache::kMax) c->plans.erase(c->plans.begin());
        c->plans.emplace_back(k, P);
    }
    return FS_OK;
}

fs_status check_device(const fs_net *net)
{
    if (net->device < 0) return fail(FS_ERR_INVALID_ARG, "net was created for planning only");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != net->device)
        return fail(FS_ERR_INVALID_ARG, "current device %d is not the net's device %d", dev, net->device);
    return FS_OK;
}

// Plan of a scan with a border mode: the mirrored modes scan the extended
// image (H + w_0 - 1) x (W + w_0 - 1), built in the workspace after the
// scan's own buffers (from byte pad_off).
fs_status border_plan(const fs_net *net, int B, int H, int W, int border, std::shared_ptr<const Plan> &PP,
                      int &He, int &We, size_t &pad_off, size_t &ws_total)
{
    if (border != BORDER_VALID && border != BORDER_REFLECT && border != BORDER_SYMMETRIC)
        return fail(FS_ERR_INVALID_ARG, "unknown border mode %d", border);
    He = H;
    We = W;
    if (border != BORDER_VALID) {
        if (B < 1 || H < 1 || W < 1) return fail(FS_ERR_SHAPE, "B, H, W must be >= 1");
        He = H + net->patch - 1;
        We = W + net->patch_x - 1;
    }
    fs_status st = get_plan(net, B, He, We, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    pad_off = P.ws_bytes;
    ws_total = P.ws_bytes;
    if (border != BORDER_VALID) {
        pad_off = align_up(P.ws_bytes, 256);
        ws_total = pad_off + (size_t)B * He * We * net->C * sizeof(float);
    }
    return FS_OK;
}

fs_status validate_scan(const fs_net *net, const float *d_image, int B, int H, int W, float *d_out,
                        void *d_ws, size_t ws_bytes, std::shared_ptr<const Plan> &PP)
{
    if (!net) return fail(FS_ERR_INVALID_ARG, "net is NULL");
    if (!d_image || !d_out) return fail(FS_ERR_INVALID_ARG, "image or output pointer is NULL");
    if (((uintptr_t)d_image & 15) || ((uintptr_t)d_out & 15))
        return fail(FS_ERR_INVALID_ARG, "image and output must be 16-byte aligned");
    fs_status st = get_plan(net, B, H, W, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    if (ws_bytes < P.ws_bytes)
        return fail(FS_ERR_WORKSPACE, "workspace of %zu bytes, the scan needs %zu", ws_bytes, P.ws_bytes);
    if (P.ws_bytes && !d_ws) return fail(FS_ERR_INVALID_ARG, "workspace pointer is NULL");
    if ((uintptr_t)d_ws & 255) return fail(FS_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    return check_device(net);
}

// A scan cut into output tiles of at most th x tw windows: the tile with
// top-left window (y0, x0) reads image rows y0 .. y0 + h + w_0 - 2 (and the
// same columns) and writes its h x w windows at (y0, x0) of the full map.
// Tiles of one shape share a plan (at most four shapes: full and last).
struct Tiled {
    int ny = 0, nx = 0, th = 0, tw = 0, rows = 0, cols = 0;
    std::shared_ptr<const Plan> shape[2][2];  // [last row of tiles][last column of tiles]
    size_t ws_bytes = 0;
    int n_launches = 0;
    double flops = 0, bytes = 0;
};

fs_status tiled_plan(const fs_net *net, int B, int H, int W, int th, int tw, Tiled &T)
{
    if (th < 1 || tw < 1) return fail(FS_ERR_INVALID_ARG, "tile sizes must be >= 1 (got %d x %d)", th, tw);
    if (B < 1 || H < net->patch || W < net->patch_x)
        return fail(FS_ERR_SHAPE, "image %dx%d (batch %d) smaller than the window %dx%d", H, W, B, net->patch,
                    net->patch_x);
    T = Tiled();
    T.ny = H - net->patch + 1;
    T.nx = W - net->patch_x + 1;
    T.th = std::min(th, T.ny);
    T.tw = std::min(tw, T.nx);
    T.rows = (T.ny + T.th - 1) / T.th;
    T.cols = (T.nx + T.tw - 1) / T.tw;
    if ((long long)T.rows * T.cols > (1 << 20)) return fail(FS_ERR_INVALID_ARG, "more than 2^20 tiles");
    for (int lr = 0; lr < 2; ++lr)
        for (int lc = 0; lc < 2; ++lc) {
            const int h = lr ? T.ny - (T.rows - 1) * T.th : T.th, w = lc ? T.nx - (T.cols - 1) * T.tw : T.tw;
            View v;
            v.img_h = H;
            v.img_w = W;
            v.out_h = T.ny;
            v.out_w = T.nx;
            fs_status st = get_plan(net, B, h + net->patch - 1, w + net->patch_x - 1, T.shape[lr][lc], &v);
            if (st != FS_OK) return st;
            T.ws_bytes = std::max(T.ws_bytes, T.shape[lr][lc]->ws_bytes);
        }
    for (int r = 0; r < T.rows; ++r)
        for (int c = 0; c < T.cols; ++c) {
            const Plan &P = *T.shape[r == T.rows - 1][c == T.cols - 1];
            T.n_launches += (int)P.launches.size();
            T.flops += P.flops;
            T.bytes += P.bytes;
        }
    return FS_OK;
}

// Launch i of plan P.  The plan is shared (cached) and left untouched: the
// launch's arguments are copied and given their buffers here.  img_off /
// out_off (floats) place a tiled scan's region in the image and the map.
hipError_t enqueue(const fs_net *net, const Plan &P, const float *d_image, float *d_out, void *d_ws,
                   hipStream_t s, int i, unsigned *dbg, int shrink_at, size_t img_off = 0, size_t out_off = 0)
{
    Launch L = P.launches[i];
    const int shrink = i == shrink_at ? 1 : 0;
    L.conv.dbg = L.pool.dbg = L.head.dbg = dbg;
    L.conv.dbg_shrink = L.pool.dbg_shrink = L.head.dbg_shrink = shrink;
    char *ws = static_cast<char *>(d_ws);
    d_image += img_off;
    d_out += out_off;
    auto ptr = [&](int which) -> void * {
        if (which == -1) return const_cast<float *>(d_image);
        if (which == 2) return d_out;
        return ws + (size_t)which * P.buf_bytes;
    };
    const char *mem = static_cast<const char *>(net->d_mem);
    if (L.type == 0) {
        const NetLayer &l = net->L[L.layer];
        L.conv.in = ptr(L.src);
        L.conv.out = ptr(L.dst);
        L.conv.w = mem + l.w_off;
        L.conv.bias = reinterpret_cast<const float *>(mem + l.b_off);
        if (L.conv.head_ncls > 0) {
            L.conv.head_w = reinterpret_cast<const float *>(mem + net->head_wp_off);
            L.conv.head_wbf = net->has_head_wbf ? mem + net->head_wbf_off : nullptr;
            L.conv.head_b = reinterpret_cast<const float *>(mem + net->head_b_off);
            L.conv.head_out = d_out;
            L.conv.out = nullptr;
        }
        if (L.direct)
            return launch_conv_direct(L.conv, reinterpret_cast<const float *>(mem + l.w32_off), net->dtype,
                                      L.in_f32, L.gx, s);
        return launch_conv(L.conv, net->dtype, L.in_f32, L.mb, L.nb, L.wn, L.wk, L.vec, L.gx, L.gy, s);
    }
    if (L.type == 1) {
        L.pool.in = ptr(L.src);
        L.pool.out = ptr(L.dst);
        return launch_pool(L.pool, net->dtype, L.in_f32, L.gx, s);
    }
    L.head.in = ptr(L.src);
    L.head.out = d_out;
    L.head.w = reinterpret_cast<const float *>(mem + net->head_w_off);
    L.head.bias = reinterpret_cast<const float *>(mem + net->head_b_off);
    return launch_head(L.head, net->dtype, L.in_f32, L.has_fc, L.gx, s);
}

}  // namespace

// ---------------------------------------------------------------------------
// C-ABI
// ---------------------------------------------------------------------------

extern "C" {

const char *fs_status_str(fs_status s)
{
    switch (s) {
    case FS_OK: return "ok";
    case FS_ERR_INVALID_ARG: return "invalid argument";
    case FS_ERR_SHAPE: return "shape not allowed";
    case FS_ERR_UNSUPPORTED: return "unsupported";
    case FS_ERR_WORKSPACE: return "workspace too small";
    case FS_ERR_OOM: return "out of device memory";
    case FS_ERR_HIP: return "HIP runtime error";
    case FS_ERR_BOUNDS: return "bounds check failed (debug library)";
    }
    return "unknown status";
}

const char *fs_last_error(void) { return g_err.c_str(); }

static fs_status net_create(const fs_layer *layers, int32_t n_layers, int32_t in_channels, int32_t patch,
                            int32_t dtype, bool upload, fs_net **out)
{
    if (!out) return fail(FS_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!layers || n_layers < 1) return fail(FS_ERR_INVALID_ARG, "no layers");
    if (in_channels < 1) return fail(FS_ERR_INVALID_ARG, "in_channels must be >= 1");
    if (dtype != FS_F32 && dtype != FS_BF16) return fail(FS_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (patch < 0) return fail(FS_ERR_INVALID_ARG, "patch must be >= 0");

    // --- validate the stack (Section 2) ---
    std::vector<NetLayer> L(n_layers);
    bool seen_fc = false;
    int c = in_channels;
    for (int i = 0; i < n_layers; ++i) {
        const fs_layer &s = layers[i];
        NetLayer &l = L[i];
        l.kind = s.kind;
        l.k = s.k;
        l.kx = s.k_x ? s.k_x : s.k;
        l.cin = s.c_in;
        l.cout = s.c_out;
        l.act = s.act;
        if (s.kind != FS_CONV && s.kind != FS_MAXPOOL && s.kind != FS_FC)
            return fail(FS_ERR_INVALID_ARG, "layer %d: unknown kind %d", i, s.kind);
        if (s.act != FS_ACT_NONE && s.act != FS_ACT_TANH && s.act != FS_ACT_SOFTMAX)
            return fail(FS_ERR_INVALID_ARG, "layer %d: unknown activation %d", i, s.act);
        if (s.act == FS_ACT_SOFTMAX && i != n_layers - 1)
            return fail(FS_ERR_SHAPE, "layer %d: softmax is allowed on the last layer only", i);
        if (s.c_in != c) return fail(FS_ERR_SHAPE, "layer %d: c_in %d, the layer below gives %d", i, s.c_in, c);
        if (s.c_in < 1 || s.c_out < 1) return fail(FS_ERR_SHAPE, "layer %d: channel counts must be >= 1", i);
        if (s.c_in > kMaxChannels || s.c_out > kMaxChannels)
            return fail(FS_ERR_UNSUPPORTED, "layer %d: more than %d channels", i, kMaxChannels);
        if (s.stride < 0 || s.stride_x < 0) return fail(FS_ERR_INVALID_ARG, "layer %d: negative stride", i);
        if (s.kind == FS_MAXPOOL) {
            if (seen_fc) return fail(FS_ERR_SHAPE, "layer %d: pooling after a fully connected layer", i);
            if (s.k < 1 || l.kx < 1) return fail(FS_ERR_SHAPE, "layer %d: pool size must be >= 1", i);
            // stride 0: the pool's own size (the paper's non-overlapping
            // pools); stride_x 0: the row stride when one is given
            l.sy = s.stride ? s.stride : l.k;
            l.sx = s.stride_x ? s.stride_x : (s.stride ? s.stride : l.kx);
            if (s.c_out != s.c_in) return fail(FS_ERR_SHAPE, "layer %d: a pool keeps the channel count", i);
            if (s.weight || s.bias) return fail(FS_ERR_INVALID_ARG, "layer %d: a pool has no weights", i);
            if (s.act != FS_ACT_NONE) return fail(FS_ERR_UNSUPPORTED, "layer %d: activation on a pool", i);
        } else {
            if (s.kind == FS_CONV && seen_fc)
                return fail(FS_ERR_SHAPE, "layer %d: convolution after a fully connected layer", i);
            if (s.stride || s.stride_x)
                return fail(FS_ERR_UNSUPPORTED, "layer %d: the method's convolutions have stride 1", i);
            if (s.kind == FS_FC) seen_fc = true;
            if (s.k < 0 || (s.k == 0 && s.kind != FS_FC)) return fail(FS_ERR_SHAPE, "layer %d: bad kernel size", i);
            if (s.k_x < 0 || (s.k == 0) != (l.kx == 0))
                return fail(FS_ERR_SHAPE, "layer %d: bad kernel columns %d", i, s.k_x);
            if (!s.weight) return fail(FS_ERR_INVALID_ARG, "layer %d: weight is NULL", i);
        }
        c = s.c_out;
    }
    // patch-level sizes: derive h_0 x w_0 when the fully connected sizes are
    // given (each axis on its own: Section 2's rectangular case)
    bool derivable = true;
    for (auto &l : L)
        if (l.kind == FS_FC && l.k == 0) derivable = false;
    int h0 = patch, w0 = patch;
    if (derivable) {
        int h = 1, w = 1;
        for (int i = n_layers - 1; i >= 0; --i) {
            h = (L[i].kind == FS_MAXPOOL) ? (h - 1) * L[i].sy + L[i].k : h + L[i].k - 1;
            w = (L[i].kind == FS_MAXPOOL) ? (w - 1) * L[i].sx + L[i].kx : w + L[i].kx - 1;
        }
        if (patch == 0) {
            h0 = h;
            w0 = w;
        } else if (patch != h || patch != w) {
            return fail(FS_ERR_SHAPE, "patch %d does not match the stack, which needs %dx%d", patch, h, w);
        }
    } else if (patch == 0) {
        return fail(FS_ERR_INVALID_ARG, "patch is 0 and a fully connected layer has k = 0");
    }
    {
        int h = h0, w = w0;
        for (int i = 0; i < n_layers; ++i) {
            NetLayer &l = L[i];
            l.h_in = h;
            l.w_in = w;
            if (l.kind == FS_MAXPOOL) {
                // Section 2.1.2: mod(w, k) = 0; with a stride s, the windows
                // at 0, s, ... must end at the map's edge: mod(w - k, s) = 0
                if (h < l.k || w < l.kx || (h - l.k) % l.sy || (w - l.kx) % l.sx)
                    return fail(FS_ERR_SHAPE, "layer %d: pool %dx%d (stride %dx%d) does not tile the map %dx%d", i,
                                l.k, l.kx, l.sy, l.sx, h, w);
                h = (h - l.k) / l.sy + 1;
                w = (w - l.kx) / l.sx + 1;
            } else {
                if (l.kind == FS_FC && l.k == 0) {
                    l.k = h;
                    l.kx = w;
                }
                if (l.kind == FS_FC && (l.k != h || l.kx != w))
                    return fail(FS_ERR_SHAPE, "layer %d: fully connected kernel %dx%d on a %dx%d map", i, l.k, l.kx,
                                h, w);
                if (l.k > h || l.kx > w)
                    return fail(FS_ERR_SHAPE, "layer %d: kernel %dx%d larger than the map %dx%d", i, l.k, l.kx, h, w);
                h -= l.k - 1;
                w -= l.kx - 1;
            }
            l.h_out = h;
            l.w_out = w;
        }
        if (h != 1 || w != 1) return fail(FS_ERR_SHAPE, "the last map is %dx%d, not 1x1", h, w);
    }

    fs_net *net = new (std::nothrow) fs_net();
    if (!net) return fail(FS_ERR_OOM, "host allocation failed");
    net->patch = h0;
    net->patch_x = w0;
    net->C = in_channels;
    net->dtype = dtype;
    net->ncls = L.back().cout;
    for (auto &l : L)
        if (l.kind == FS_MAXPOOL) {
            net->pool_k.push_back(l.sy);
            net->pool_kx.push_back(l.sx);
            net->S *= l.sy;
            net->Sx *= l.sx;
            net->F *= l.sy * l.sx;
        }
    if (net->S > kMaxAxis || net->Sx > kMaxAxis) {
        delete net;
        return fail(FS_ERR_UNSUPPORTED, "pool sizes multiply to %dx%d > %d per axis", net->S, net->Sx, kMaxAxis);
    }
    if (net->ncls > kMaxHeadClasses) {
        delete net;
        return fail(FS_ERR_UNSUPPORTED, "%d outputs; at most %d supported", net->ncls, kMaxHeadClasses);
    }
    const NetLayer &last = L.back();
    net->head_fc = last.kind != FS_MAXPOOL && last.k == 1 && last.kx == 1 && last.cin * last.cout <= kMaxHeadWeights;
    net->head_cin = net->head_fc ? last.cin : 0;

    // --- pack parameters into one device block ---
    std::vector<uint8_t> blob;
    auto push = [&](const void *p, size_t n) {
        const size_t off = align_up(blob.size(), 256);
        blob.resize(off + n);
        std::memcpy(blob.data() + off, p, n);
        return off;
    };
    const int KSTEP = kstep_of(dtype);
    for (int i = 0; i < n_layers; ++i) {
        NetLayer &l = L[i];
        if (l.kind == FS_MAXPOOL) continue;
        const fs_layer &s = layers[i];
        std::vector<float> bias(l.cout, 0.f);
        if (s.bias) std::memcpy(bias.data(), s.bias, sizeof(float) * l.cout);
        if (i == n_layers - 1 && net->head_fc) {
            std::vector<float> w((size_t)l.cout * l.cin);
            std::memcpy(w.data(), s.weight, sizeof(float) * w.size());
            net->head_w_off = push(w.data(), w.size() * 4);
            net->head_b_off = push(bias.data(), bias.size() * 4);
            // the same weights over the previous layer's (block, row) order,
            // for the head fused into that layer's epilogue
            if (i >= 1 && L[i - 1].kind != FS_MAXPOOL && L[i - 1].nbt > 0) {
                const NetLayer &pl = L[i - 1];
                // at least kMaxFusedClasses rows (zero past the classes)
                std::vector<float> wp((size_t)std::max(l.cout, kMaxFusedClasses) * pl.nbt * 16, 0.f);
                for (int c = 0; c < l.cout; ++c)
                    for (int r = 0; r < pl.nbt * 16; ++r) {
                        const int ci = chan_of(pl, dtype, r / 16, r % 16);
                        if (ci < l.cin) wp[(size_t)c * pl.nbt * 16 + r] = w[(size_t)c * l.cin + ci];
                    }
                net->head_wp_off = push(wp.data(), wp.size() * 4);
                if (dtype == DT_BF16 && pl.nb % 2 == 0) {
                    std::vector<uint16_t> wb((size_t)pl.nbt / 2 * 64 * 8, 0);
                    for (int P = 0; P < pl.nbt / 2; ++P)
                        for (int lane = 0; lane < 64; ++lane)
                            for (int e = 0; e < 8; ++e) {
                                const int c = lane % 16, ci = 32 * P + 8 * (lane / 16) + e;
                                if (c < l.cout && ci < l.cin)
                                    wb[((size_t)P * 64 + lane) * 8 + e] = host_f2bf(w[(size_t)c * l.cin + ci]);
                            }
                    net->head_wbf_off = push(wb.data(), wb.size() * 2);
                    net->has_head_wbf = true;
                }
            }
            continue;
        }
        // the layer that reads the float32 image of a bf16 net converts while
        // staging, which the gather path does
        l.vec = (l.cin % KSTEP) == 0 && !(dtype == FS_BF16 && i == 0);
        const int nbt0 = (l.cout + 15) / 16;
        choose_channel_tile(nbt0, l.vec, &l.nb, &l.wn);
        // narrow channel tiles with a long K walk: two waves split K so each
        // wave owns 4 pixel blocks (more products per operand load, measured
        // faster on the 48 -> 48 layers of N4) without a larger LDS window
        l.wk = (l.vec && l.wn == 1 && l.nb == 3 && l.k * l.kx * l.cin >= 16 * 16) ? 2 : 1;
        tile_override(i, nullptr, &l.nb, &l.wn, nullptr, &l.wk);
        bool any = false;
        for (int mb : {1, 2, 4, 8}) any = any || conv_tile_supported(mb, l.nb, l.wn, l.wk, l.vec);
        if (!any) {
            delete net;
            return fail(FS_ERR_UNSUPPORTED, "layer %d: no convolution tile with %d x %d channel blocks", i,
                        l.nb, l.wn);
        }
        const int grp = l.nb * l.wn;
        l.nbt = (nbt0 + grp - 1) / grp * grp;
        l.ksteps = l.vec ? l.k * l.kx * (l.cin / KSTEP) : (l.k * l.kx * l.cin + KSTEP - 1) / KSTEP;
        if (l.ksteps < l.wk) {  // every K-splitting wave needs at least one step
            delete net;
            return fail(FS_ERR_UNSUPPORTED, "layer %d: %d K steps cannot be split over %d waves", i, l.ksteps, l.wk);
        }
        std::vector<uint8_t> pw;
        pack_conv_weights(l, s.weight, dtype, pw);
        l.w_off = push(pw.data(), pw.size());
        // bias in (block, row) order
        std::vector<float> bp((size_t)l.nbt * 16, 0.f);
        for (int r = 0; r < l.nbt * 16; ++r) {
            const int co = chan_of(l, dtype, r / 16, r % 16);
            if (co < l.cout) bp[r] = bias[co];
        }
        l.b_off = push(bp.data(), bp.size() * 4);
        if (!l.vec && conv_direct_supported(l.cin, l.k * l.kx, l.cout)) {
            // [rows][KP] copy for the direct kernel, K index (dy * k_x + dx) * c_in + ci,
            // then the biases in channel order
            const int kp = conv_direct_kp(l.cin, l.k * l.kx);
            const int rows = (l.cout + 7) / 8 * 8;
            std::vector<float> wd((size_t)rows * kp + l.cout, 0.f);
            std::copy(bias.begin(), bias.end(), wd.begin() + (size_t)rows * kp);
            for (int co = 0; co < l.cout; ++co)
                for (int dy = 0; dy < l.k; ++dy)
                    for (int dx = 0; dx < l.kx; ++dx)
                        for (int ci = 0; ci < l.cin; ++ci) {
                            float v = s.weight[(((size_t)co * l.cin + ci) * l.k + dy) * l.kx + dx];
                            if (dtype == FS_BF16) {
                                const uint32_t u = (uint32_t)host_f2bf(v) << 16;
                                std::memcpy(&v, &u, 4);
                            }
                            wd[(size_t)co * kp + (dy * l.kx + dx) * l.cin + ci] = v;
                        }
            l.has_w32 = true;
            l.w32_off = push(wd.data(), wd.size() * 4);
        }
    }
    if (!net->head_fc) {  // the head still takes a (unused) bias pointer
        std::vector<float> z(kMaxHeadClasses, 0.f);
        net->head_w_off = push(z.data(), z.size() * 4);
        net->head_b_off = push(z.data(), z.size() * 4);
    }
    net->L = L;
    net->plans = new (std::nothrow) PlanCache();  // (without one, every scan plans afresh)
    if (!upload) {  // planning-only handle: no device memory
        net->device = -1;
        *out = net;
        return FS_OK;
    }
    hipError_t e = hipGetDevice(&net->device);
    if (e != hipSuccess) {
        delete net;
        return hip_fail(e, "hipGetDevice");
    }
    {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, net->device) == hipSuccess && n > 0)
            net->ncu = n;
    }
    {
        // set-up of the no-allocation entry point on this device: its scratch
        // address (a failure here is reported by fs_scan_noalloc itself)
        void *p = nullptr;
        if (scratch_on(net->device, &p) != FS_OK) g_err.clear();
    }
    net->mem_bytes = blob.size();
    e = hipMalloc(&net->d_mem, blob.size());
    if (e != hipSuccess) {
        delete net;
        return fail(FS_ERR_OOM, "hipMalloc(%zu): %s", blob.size(), hipGetErrorString(e));
    }
    e = hipMemcpy(net->d_mem, blob.data(), blob.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(net->d_mem);
        delete net;
        return hip_fail(e, "hipMemcpy (weights)");
    }
    *out = net;
    return FS_OK;
}

fs_status fs_net_create(const fs_layer *layers, int32_t n_layers, int32_t in_channels, int32_t patch,
                        int32_t dtype, fs_net **out)
{
    return net_create(layers, n_layers, in_channels, patch, dtype, true, out);
}

fs_status fs_net_create_plan_only(const fs_layer *layers, int32_t n_layers, int32_t in_channels,
                                  int32_t patch, int32_t dtype, fs_net **out)
{
    return net_create(layers, n_layers, in_channels, patch, dtype, false, out);
}

void fs_net_destroy(fs_net *net)
{
    if (!net) return;
    if (net->d_mem) (void)hipFree(net->d_mem);
    delete net;
}

fs_status fs_net_query(const fs_net *net, fs_net_info *out)
{
    if (!net || !out) return fail(FS_ERR_INVALID_ARG, "NULL argument");
    out->patch = net->patch;
    out->in_channels = net->C;
    out->n_classes = net->ncls;
    out->n_layers = (int)net->L.size();
    out->n_pools = (int)net->pool_k.size();
    out->stride = net->S;
    out->n_fragments = net->F;
    out->dtype = net->dtype;
    out->patch_x = net->patch_x;
    out->stride_x = net->Sx;
    return FS_OK;
}

fs_status fs_scan_plan_tiled(const fs_net *net, int32_t B, int32_t H, int32_t W, int32_t tile_h, int32_t tile_w,
                             fs_plan_info *out)
{
    if (!net || !out) return fail(FS_ERR_INVALID_ARG, "NULL argument");
    Tiled T;
    fs_status st = tiled_plan(net, B, H, W, tile_h, tile_w, T);
    if (st != FS_OK) return st;
    out->batch = B;
    out->out_h = T.ny;
    out->out_w = T.nx;
    out->n_launches = T.n_launches;
    out->workspace_bytes = T.ws_bytes;
    out->flops = T.flops;
    out->min_bytes = T.bytes;
    return FS_OK;
}

fs_status fs_scan_tiled(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W, int32_t tile_h,
                        int32_t tile_w, float *d_out, void *d_workspace, size_t workspace_bytes, void *stream)
{
    if (!net) return fail(FS_ERR_INVALID_ARG, "net is NULL");
    if (!d_image || !d_out) return fail(FS_ERR_INVALID_ARG, "image or output pointer is NULL");
    if (((uintptr_t)d_image & 15) || ((uintptr_t)d_out & 15))
        return fail(FS_ERR_INVALID_ARG, "image and output must be 16-byte aligned");
    Tiled T;
    fs_status st = tiled_plan(net, B, H, W, tile_h, tile_w, T);
    if (st != FS_OK) return st;
    if (workspace_bytes < T.ws_bytes)
        return fail(FS_ERR_WORKSPACE, "workspace of %zu bytes, the tiled scan needs %zu", workspace_bytes, T.ws_bytes);
    if (T.ws_bytes && !d_workspace) return fail(FS_ERR_INVALID_ARG, "workspace pointer is NULL");
    if ((uintptr_t)d_workspace & 255) return fail(FS_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    st = check_device(net);
    if (st != FS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned *dbg = nullptr;
    st = dbg_begin(s, &dbg);
    if (st != FS_OK) return st;
    const int shrink_at = dbg_shrink_at();
    for (int r = 0; r < T.rows; ++r)
        for (int c = 0; c < T.cols; ++c) {
            const Plan &P = *T.shape[r == T.rows - 1][c == T.cols - 1];
            const size_t y0 = (size_t)r * T.th, x0 = (size_t)c * T.tw;
            const size_t img_off = (y0 * W + x0) * net->C, out_off = (y0 * T.nx + x0) * net->ncls;
            for (int i = 0; i < (int)P.launches.size(); ++i) {
                hipError_t e = enqueue(net, P, d_image, d_out, d_workspace, s, i, dbg, shrink_at, img_off, out_off);
                if (e != hipSuccess)
                    return fail(FS_ERR_HIP, "tile (%d, %d) launch %d (%s): %s", r, c, i, P.launches[i].name.c_str(),
                                hipGetErrorString(e));
            }
        }
    return dbg_end(s, dbg);
}

fs_status fs_scan_plan(const fs_net *net, int32_t B, int32_t H, int32_t W, fs_plan_info *out)
{
    if (!net || !out) return fail(FS_ERR_INVALID_ARG, "NULL argument");
    std::shared_ptr<const Plan> PP;
    fs_status st = get_plan(net, B, H, W, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    out->batch = B;
    out->out_h = P.ny;
    out->out_w = P.nx;
    out->n_launches = (int)P.launches.size();
    out->workspace_bytes = P.ws_bytes;
    out->flops = P.flops;
    out->min_bytes = P.bytes;
    return FS_OK;
}

fs_status fs_scan_plan_border(const fs_net *net, int32_t B, int32_t H, int32_t W, int32_t border,
                              fs_plan_info *out)
{
    if (!net || !out) return fail(FS_ERR_INVALID_ARG, "NULL argument");
    std::shared_ptr<const Plan> PP;
    int He, We;
    size_t pad_off, ws_total;
    fs_status st = border_plan(net, B, H, W, border, PP, He, We, pad_off, ws_total);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    out->batch = B;
    out->out_h = P.ny;
    out->out_w = P.nx;
    out->n_launches = (int)P.launches.size() + (border != BORDER_VALID);
    out->workspace_bytes = ws_total;
    out->flops = P.flops;
    out->min_bytes = P.bytes + (border != BORDER_VALID ? 2.0 * B * He * We * net->C * sizeof(float) : 0.0);
    return FS_OK;
}

fs_status fs_scan_border(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W, int32_t border,
                         float *d_out, void *d_workspace, size_t workspace_bytes, void *stream)
{
    if (!net) return fail(FS_ERR_INVALID_ARG, "net is NULL");
    if (!d_image || !d_out) return fail(FS_ERR_INVALID_ARG, "image or output pointer is NULL");
    if (((uintptr_t)d_image & 15) || ((uintptr_t)d_out & 15))
        return fail(FS_ERR_INVALID_ARG, "image and output must be 16-byte aligned");
    std::shared_ptr<const Plan> PP;
    int He, We;
    size_t pad_off, ws_total;
    fs_status st = border_plan(net, B, H, W, border, PP, He, We, pad_off, ws_total);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    if (workspace_bytes < ws_total)
        return fail(FS_ERR_WORKSPACE, "workspace of %zu bytes, the scan needs %zu", workspace_bytes, ws_total);
    if (ws_total && !d_workspace) return fail(FS_ERR_INVALID_ARG, "workspace pointer is NULL");
    if ((uintptr_t)d_workspace & 255) return fail(FS_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    st = check_device(net);
    if (st != FS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned *dbg = nullptr;
    st = dbg_begin(s, &dbg);
    if (st != FS_OK) return st;
    const int shrink_at = dbg_shrink_at();
    const float *img = d_image;
    if (border != BORDER_VALID) {
        float *pad = reinterpret_cast<float *>(static_cast<char *>(d_workspace) + pad_off);
        const int p0y = (net->patch - 1) / 2, p0x = (net->patch_x - 1) / 2;
        hipError_t e = launch_mirror_pad(d_image, pad, B, H, W, net->C, p0y, p0x, He, We, border, dbg,
                                         shrink_at == -2 ? 1 : 0, s);
        if (e != hipSuccess) return fail(FS_ERR_HIP, "mirror pad: %s", hipGetErrorString(e));
        img = pad;
    }
    for (int i = 0; i < (int)P.launches.size(); ++i) {
        hipError_t e = enqueue(net, P, img, d_out, d_workspace, s, i, dbg, shrink_at);
        if (e != hipSuccess) return fail(FS_ERR_HIP, "launch %d (%s): %s", i, P.launches[i].name.c_str(),
                                         hipGetErrorString(e));
    }
    return dbg_end(s, dbg);
}

fs_status fs_scan_launches(const fs_net *net, int32_t B, int32_t H, int32_t W, fs_launch_info *h_out,
                           int32_t capacity)
{
    if (!net || (!h_out && capacity > 0) || capacity < 0) return fail(FS_ERR_INVALID_ARG, "bad argument");
    std::shared_ptr<const Plan> PP;
    fs_status st = get_plan(net, B, H, W, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    const int n = std::min<int>(capacity, (int)P.launches.size());
    for (int i = 0; i < n; ++i) {
        const Launch &L = P.launches[i];
        fs_launch_info &o = h_out[i];
        std::memset(&o, 0, sizeof o);
        o.layer = L.layer;
        o.n_layers = L.n_layers;
        o.kind = L.type;
        o.fragments = L.frags;
        o.out_pixels = L.out_pixels;
        o.flops = L.flops;
        o.bytes = L.bytes;
        o.grid = L.gx * L.gy;
        o.block = 256;
        std::snprintf(o.name, sizeof o.name, "%s", L.name.c_str());
        if (L.type == 0 && !L.direct) {
            o.lds_bytes = L.conv.lds_bytes;
            if (net->ncu > 0)
                o.per_cu = conv_blocks_per_cu(net->dtype, L.in_f32, L.mb, L.nb, L.wn, L.wk, L.vec, L.conv.run,
                                              L.conv.lds_bytes);
        }
    }
    return FS_OK;
}

fs_status fs_scan(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W, float *d_out,
                  void *d_workspace, size_t workspace_bytes, void *stream)
{
    std::shared_ptr<const Plan> PP;
    fs_status st = validate_scan(net, d_image, B, H, W, d_out, d_workspace, workspace_bytes, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned *dbg = nullptr;
    st = dbg_begin(s, &dbg);
    if (st != FS_OK) return st;
    const int shrink_at = dbg_shrink_at();
    for (int i = 0; i < (int)P.launches.size(); ++i) {
        hipError_t e = enqueue(net, P, d_image, d_out, d_workspace, s, i, dbg, shrink_at);
        if (e != hipSuccess) return fail(FS_ERR_HIP, "launch %d (%s): %s", i, P.launches[i].name.c_str(),
                                         hipGetErrorString(e));
    }
    return dbg_end(s, dbg);
}

fs_status fs_scan_noalloc(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W, float *d_out,
                          void *stream)
{
    if (!net) return fail(FS_ERR_INVALID_ARG, "net is NULL");
    if (!d_image || !d_out) return fail(FS_ERR_INVALID_ARG, "image or output pointer is NULL");
    if (((uintptr_t)d_image & 15) || ((uintptr_t)d_out & 15))
        return fail(FS_ERR_INVALID_ARG, "image and output must be 16-byte aligned");
    std::shared_ptr<const Plan> PP;
    fs_status st = get_plan(net, B, H, W, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    if (P.ws_bytes > FS_NOALLOC_SCRATCH_BYTES)
        return fail(FS_ERR_WORKSPACE, "the scan needs %zu bytes of workspace; fs_scan_noalloc has %zu (use fs_scan)",
                    P.ws_bytes, (size_t)FS_NOALLOC_SCRATCH_BYTES);
    st = check_device(net);
    if (st != FS_OK) return st;
    void *ws = nullptr;
    st = scratch_on(net->device, &ws);
    if (st != FS_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    unsigned *dbg = nullptr;
    st = dbg_begin(s, &dbg);
    if (st != FS_OK) return st;
    const int shrink_at = dbg_shrink_at();
    for (int i = 0; i < (int)P.launches.size(); ++i) {
        hipError_t e = enqueue(net, P, d_image, d_out, ws, s, i, dbg, shrink_at);
        if (e != hipSuccess) return fail(FS_ERR_HIP, "launch %d (%s): %s", i, P.launches[i].name.c_str(),
                                         hipGetErrorString(e));
    }
    return dbg_end(s, dbg);
}

fs_status fs_scan_profile(const fs_net *net, const float *d_image, int32_t B, int32_t H, int32_t W,
                          float *d_out, void *d_workspace, size_t workspace_bytes, void *stream, int32_t reps,
                          float *h_launch_ms, int32_t capacity)
{
    if (reps < 1 || capacity < 0 || (!h_launch_ms && capacity > 0))
        return fail(FS_ERR_INVALID_ARG, "bad reps / output");
    std::shared_ptr<const Plan> PP;
    fs_status st = validate_scan(net, d_image, B, H, W, d_out, d_workspace, workspace_bytes, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int n = (int)P.launches.size();
    // Launch i runs `reps` times back to back between two events.  Every
    // launch reads one buffer and writes another (or the output), so a
    // repetition recomputes the same values and the launches that follow see
    // exactly what a plain scan leaves them.
    unsigned *dbg = nullptr;
    st = dbg_begin(s, &dbg);
    if (st != FS_OK) return st;
    const int shrink_at = dbg_shrink_at();
    std::vector<hipEvent_t> ev((size_t)n * 2, nullptr);
    hipError_t e = hipSuccess;
    for (auto &x : ev) {
        e = hipEventCreate(&x);
        if (e != hipSuccess) break;
    }
    for (int i = 0; i < n && e == hipSuccess; ++i) {
        e = hipEventRecord(ev[2 * i], s);
        for (int r = 0; r < reps && e == hipSuccess; ++r)
            e = enqueue(net, P, d_image, d_out, d_workspace, s, i, dbg, shrink_at);
        if (e == hipSuccess) e = hipEventRecord(ev[2 * i + 1], s);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    std::vector<double> ms_i(n, 0.0);
    for (int i = 0; i < n && e == hipSuccess; ++i) {
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, ev[2 * i], ev[2 * i + 1]);
        ms_i[i] = ms;
    }
    for (auto &x : ev)
        if (x) (void)hipEventDestroy(x);
    if (e != hipSuccess) return hip_fail(e, "profiled scan");
    for (int i = 0; i < std::min(n, (int)capacity); ++i) h_launch_ms[i] = (float)(ms_i[i] / reps);
    return dbg_end(s, dbg);
}

fs_status fs_fragment_table(const fs_net *net, int32_t H, int32_t W, int32_t *h_out, size_t capacity,
                            size_t *n_needed)
{
    if (!net) return fail(FS_ERR_INVALID_ARG, "net is NULL");
    std::shared_ptr<const Plan> PP;
    fs_status st = get_plan(net, 1, H, W, PP);  // (validates the size)
    if (st != FS_OK) return st;
    const int np = (int)net->pool_k.size();
    const size_t rec = 5 + 2 * (size_t)np;
    const size_t need = rec * net->F;
    if (n_needed) *n_needed = need;
    if (!h_out) return FS_OK;
    // final per-axis sizes: replay the size recursion on one axis table each
    std::vector<int> ey{H}, ex{W};
    for (const NetLayer &l : net->L) {
        if (l.kind == FS_MAXPOOL) {
            std::vector<int> ny, nx;
            for (size_t i = 0; i < ey.size(); ++i)
                for (int o = 0; o < l.sy; ++o) ny.push_back(std::max(ey[i] - o - l.k + l.sy, 0) / l.sy);
            for (size_t i = 0; i < ex.size(); ++i)
                for (int o = 0; o < l.sx; ++o) nx.push_back(std::max(ex[i] - o - l.kx + l.sx, 0) / l.sx);
            ey.swap(ny);
            ex.swap(nx);
        } else {
            for (auto &v : ey) v = std::max(v - (l.k - 1), 0);
            for (auto &v : ex) v = std::max(v - (l.kx - 1), 0);
        }
    }
    std::vector<int32_t> r(rec);
    for (int f = 0; f < net->F; ++f) {
        // digits of f, first pool most significant: d_m = o_y * kx_m + o_x
        std::vector<int> ox(np), oy(np);
        int rest = f;
        for (int m = np - 1; m >= 0; --m) {
            const int ky = net->pool_k[m], kx = net->pool_kx[m];
            const int d = rest % (ky * kx);
            rest /= ky * kx;
            ox[m] = d % kx;
            oy[m] = d / kx;
        }
        int fy = 0, fx = 0, Y0 = 0, X0 = 0, Sy = 1, Sx = 1;
        for (int m = 0; m < np; ++m) {
            const int ky = net->pool_k[m], kx = net->pool_kx[m];
            fy = fy * ky + oy[m];
            fx = fx * kx + ox[m];
            Y0 += oy[m] * Sy;
            X0 += ox[m] * Sx;
            Sy *= ky;
            Sx *= kx;
        }
        r[0] = f;
        r[1] = ey[fy];
        r[2] = ex[fx];
        r[3] = Y0;
        r[4] = X0;
        for (int m = 0; m < np; ++m) {
            r[5 + 2 * m] = ox[m];
            r[6 + 2 * m] = oy[m];
        }
        const size_t base = (size_t)f * rec;
        for (size_t j = 0; j < rec && base + j < capacity; ++j) h_out[base + j] = r[j];
    }
    return FS_OK;
}

fs_status fs_reassembly_index(const fs_net *net, int32_t H, int32_t W, int32_t *h_out, size_t capacity,
                              size_t *n_needed)
{
    if (!net) return fail(FS_ERR_INVALID_ARG, "net is NULL");
    std::shared_ptr<const Plan> PP;
    fs_status st = get_plan(net, 1, H, W, PP);
    if (st != FS_OK) return st;
    const Plan &P = *PP;
    const size_t need = (size_t)3 * P.ny * P.nx;
    if (n_needed) *n_needed = need;
    if (!h_out) return FS_OK;
    const int np = (int)net->pool_k.size();
    for (int Y = 0; Y < P.ny; ++Y)
        for (int X = 0; X < P.nx; ++X) {
            int f = 0, ry = Y, rx = X;
            for (int m = 0; m < np; ++m) {
                const int ky = net->pool_k[m], kx = net->pool_kx[m];
                f = f * ky * kx + (ry % ky) * kx + (rx % kx);
                ry /= ky;
                rx /= kx;
            }
            const size_t base = ((size_t)Y * P.nx + X) * 3;
            const int32_t v[3] = {f, ry, rx};
            for (int j = 0; j < 3 && base + j < capacity; ++j) h_out[base + j] = v[j];
        }
    return FS_OK;
}

}  // extern "C"
