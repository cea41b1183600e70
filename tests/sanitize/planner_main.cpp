// Host-side driver for the sanitizer build of the library's planner: it runs
// every planning-only path of the C-ABI (net validation and weight packing,
// scan plans, per-launch descriptions, fragment tables, reassembly indices,
// tiled and mirrored-border plans, and the argument checks of the scan entry
// points, which return before any device work) on the workload nets and on
// seeded random stacks.  Built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code only; no GPU is touched.
// Exit status 0 when every call behaved as expected.
#include "fragscan.h"

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

namespace {

int g_fail = 0;

void expect(bool ok, const char *what)
{
    if (!ok) {
        std::fprintf(stderr, "FAILED: %s (%s)\n", what, fs_last_error());
        ++g_fail;
    }
}

struct Spec {
    int kind, k, kx, cin, cout, act;
};

// Plan-only net from layer specs with seeded weights; nullptr on failure.
fs_net *make_net(const std::vector<Spec> &spec, int c0, int dtype, std::mt19937 &rng, fs_status *st_out = nullptr)
{
    std::normal_distribution<float> nd(0.f, 0.1f);
    std::vector<std::vector<float>> w(spec.size()), b(spec.size());
    std::vector<fs_layer> L(spec.size());
    for (size_t i = 0; i < spec.size(); ++i) {
        const Spec &s = spec[i];
        L[i].kind = s.kind;
        L[i].k = s.k;
        L[i].k_x = s.kx;
        L[i].c_in = s.cin;
        L[i].c_out = s.cout;
        L[i].act = s.act;
        if (s.kind != FS_MAXPOOL) {
            const int ky = s.k, kx = s.kx ? s.kx : ky;
            w[i].resize((size_t)s.cout * s.cin * ky * kx);
            for (auto &v : w[i]) v = nd(rng);
            b[i].resize(s.cout);
            for (auto &v : b[i]) v = nd(rng);
            L[i].weight = w[i].data();
            L[i].bias = b[i].data();
        }
    }
    fs_net *net = nullptr;
    fs_status st = fs_net_create_plan_only(L.data(), (int)L.size(), c0, 0, dtype, &net);
    if (st_out) *st_out = st;
    return st == FS_OK ? net : nullptr;
}

void exercise(fs_net *net, int B, int H, int W)
{
    fs_net_info info;
    expect(fs_net_query(net, &info) == FS_OK, "query");
    fs_plan_info p;
    if (fs_scan_plan(net, B, H, W, &p) != FS_OK) return;  // e.g. an image below the window
    std::vector<fs_launch_info> li(p.n_launches);
    expect(fs_scan_launches(net, B, H, W, li.data(), (int)li.size()) == FS_OK, "launches");
    size_t need = 0;
    expect(fs_fragment_table(net, H, W, nullptr, 0, &need) == FS_OK, "table size");
    std::vector<int32_t> tab(need);
    expect(fs_fragment_table(net, H, W, tab.data(), tab.size(), nullptr) == FS_OK, "table");
    // a short buffer is filled up to its capacity only
    if (need > 3) expect(fs_fragment_table(net, H, W, tab.data(), need - 3, nullptr) == FS_OK, "short table");
    expect(fs_reassembly_index(net, H, W, nullptr, 0, &need) == FS_OK, "index size");
    std::vector<int32_t> idx(need);
    expect(fs_reassembly_index(net, H, W, idx.data(), idx.size(), nullptr) == FS_OK, "index");
    fs_plan_info t;
    (void)fs_scan_plan_tiled(net, B, H, W, 7, 11, &t);
    (void)fs_scan_plan_tiled(net, B, H, W, 1, 1 << 20, &t);
    for (int border = 0; border < 4; ++border) (void)fs_scan_plan_border(net, B, H, W, border, &t);
    // argument checks of the scan entry points: refused before any device work
    void *img = reinterpret_cast<void *>(uintptr_t(1) << 20), *out = reinterpret_cast<void *>(uintptr_t(2) << 20);
    void *ws = reinterpret_cast<void *>(uintptr_t(4) << 20);
    const float *fimg = static_cast<const float *>(img);
    float *fout = static_cast<float *>(out);
    expect(fs_scan(net, fimg, B, H, W, fout, ws, p.workspace_bytes, nullptr) == FS_ERR_INVALID_ARG,
           "planning-only scan refused");
    expect(fs_scan(net, fimg + 1, B, H, W, fout, ws, p.workspace_bytes, nullptr) == FS_ERR_INVALID_ARG,
           "misaligned image");
    expect(fs_scan(net, fimg, B, H, W, fout, ws, p.workspace_bytes ? p.workspace_bytes - 1 : 0, nullptr) !=
               FS_OK, "small workspace");
    expect(fs_scan_noalloc(net, fimg, B, H, W, fout, nullptr) != FS_OK, "planning-only noalloc refused");
    expect(fs_scan_tiled(net, fimg, B, H, W, 5, 5, fout, ws, (size_t)1 << 40, nullptr) != FS_OK,
           "planning-only tiled refused");
    float ms[4];
    expect(fs_scan_profile(net, fimg, B, H, W, fout, ws, p.workspace_bytes, nullptr, 1, ms, 4) != FS_OK,
           "planning-only profile refused");
}

}  // namespace

int main()
{
    std::mt19937 rng(1302);
    const int T = FS_ACT_TANH, N = FS_ACT_NONE, S = FS_ACT_SOFTMAX;
    // net N4 (Table 1) and the other workload nets
    const std::vector<Spec> n4 = {{0, 4, 0, 1, 48, T},  {1, 2, 0, 48, 48, N}, {0, 5, 0, 48, 48, T},
                                  {1, 2, 0, 48, 48, N}, {0, 4, 0, 48, 48, T}, {1, 2, 0, 48, 48, N},
                                  {0, 4, 0, 48, 48, T}, {1, 2, 0, 48, 48, N}, {2, 3, 0, 48, 200, T},
                                  {2, 1, 0, 200, 2, S}};
    const std::vector<Spec> mixed = {{0, 3, 0, 3, 32, N},  {0, 3, 0, 32, 32, T}, {1, 3, 0, 32, 32, N},
                                     {0, 4, 0, 32, 64, T}, {1, 2, 0, 64, 64, N}, {0, 3, 0, 64, 64, T},
                                     {1, 2, 0, 64, 64, N}, {2, 3, 0, 64, 128, T}, {2, 1, 0, 128, 4, S}};
    const std::vector<Spec> rect = {{0, 3, 2, 3, 32, T}, {1, 2, 3, 32, 32, N}, {0, 2, 3, 32, 48, T},
                                    {1, 3, 2, 48, 48, N}, {2, 2, 3, 48, 16, T}, {2, 1, 1, 16, 2, S}};
    for (int dtype = 0; dtype < 2; ++dtype) {
        fs_net *a = make_net(n4, 1, dtype, rng);
        expect(a != nullptr, "N4");
        if (a) {
            for (int s : {95, 96, 140, 512, 1024}) exercise(a, s == 1024 ? 8 : 1, s, s + 7);
            exercise(a, 1, 94, 94);
            exercise(a, 1, 95, 65536);
            fs_net_destroy(a);
        }
        fs_net *m = make_net(mixed, 3, dtype, rng);
        expect(m != nullptr, "mixed");
        if (m) {
            for (int s : {61, 62, 130, 1536}) exercise(m, 1, s, s);
            fs_net_destroy(m);
        }
        fs_net *r = make_net(rect, 3, dtype, rng);
        expect(r != nullptr, "rect");
        if (r) {
            for (int s : {25, 26, 60, 300}) exercise(r, 2, s, s + 3);
            fs_net_destroy(r);
        }
    }
    // random stacks, valid or not (rejected ones must fail cleanly)
    std::uniform_int_distribution<int> u(0, 1 << 30);
    int made = 0;
    for (int n = 0; n < 300; ++n) {
        std::vector<Spec> s;
        int c = 1 + u(rng) % 20, c0 = c;
        const int nb = 1 + u(rng) % 5;
        for (int i = 0; i < nb; ++i) {
            if (u(rng) % 2) {
                s.push_back({1, 1 + u(rng) % 3, u(rng) % 2 ? 0 : 1 + u(rng) % 3, c, c, N});
            } else {
                const int co = 1 + u(rng) % 40;
                s.push_back({0, 1 + u(rng) % 4, u(rng) % 2 ? 0 : 1 + u(rng) % 4, c, co, u(rng) % 2 ? T : N});
                c = co;
            }
        }
        const int hid = 1 + u(rng) % 30;
        s.push_back({2, 1 + u(rng) % 3, u(rng) % 2 ? 0 : 1 + u(rng) % 3, c, hid, T});
        s.push_back({2, 1, 0, hid, 2 + u(rng) % 3, S});
        fs_status st;
        fs_net *net = make_net(s, c0, u(rng) % 2, rng, &st);
        expect(net != nullptr || st == FS_ERR_SHAPE || st == FS_ERR_UNSUPPORTED || st == FS_ERR_INVALID_ARG,
               "random net status");
        if (!net) continue;
        ++made;
        fs_net_info info;
        fs_net_query(net, &info);
        for (int e : {0, 3, 40}) exercise(net, 1 + u(rng) % 2, info.patch + e, info.patch_x + e + u(rng) % 9);
        fs_net_destroy(net);
    }
    std::printf("sanitizer planner run: %d random nets planned, %d failures\n", made, g_fail);
    return g_fail ? 1 : 0;
}
