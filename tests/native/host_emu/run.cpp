// Runs the fp32 training forward and backward of one problem through the C ABI on the host
// emulation, with every buffer an exact-size heap allocation (AddressSanitizer reports any
// access outside), and writes inputs and outputs as raw float32 files for the test to compare
// with the oracle.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>

#include "fla_swin.h"

extern int emu_kernel_args;
extern int emu_fail_launch;

static float* alloc_random(size_t n, std::mt19937& g) {
    float* p = static_cast<float*>(std::aligned_alloc(16, ((n * 4 + 15) / 16) * 16));
    std::normal_distribution<float> d(0.f, 1.f);
    for (size_t i = 0; i < n; ++i) p[i] = d(g);
    return p;
}

static void dump(const char* dir, const char* name, const float* p, size_t n) {
    char path[1024];
    std::snprintf(path, sizeof path, "%s/%s.f32", dir, name);
    FILE* f = std::fopen(path, "wb");
    std::fwrite(p, 4, n, f);
    std::fclose(f);
}

// Cycle-scan through the C ABI: run cycle B L d N repeats outdir
static int run_cycle(int argc, char** argv) {
    if (argc != 8) {
        std::fprintf(stderr, "usage: run cycle B L d N repeats outdir\n");
        return 2;
    }
    const int B = std::atoi(argv[2]), L = std::atoi(argv[3]), d = std::atoi(argv[4]), N = std::atoi(argv[5]);
    const int r = std::atoi(argv[6]);
    const char* dir = argv[7];
    const size_t nx = (size_t)B * L * d, nb = (size_t)B * L * N, na = (size_t)d * N;
    std::mt19937 g(4321);
    float* x = alloc_random(nx, g);
    float* delta = alloc_random(nx, g);
    float* A = alloc_random(na, g);
    float* Bm = alloc_random(nb, g);
    float* Cm = alloc_random(nb, g);
    float* y = alloc_random(nx, g);
    for (size_t i = 0; i < nx; ++i) delta[i] = std::log1p(std::exp(delta[i] - 2.f));   // positive steps
    for (size_t i = 0; i < na; ++i) A[i] = -0.25f - std::fabs(A[i]);                   // negative diagonal
    size_t nws = 0;
    if (fla_cycle_scan_workspace(B, L, d, N, r, &nws) != 0) return 1;
    void* ws = std::aligned_alloc(16, ((nws + 15) / 16) * 16);
    emu_kernel_args = 2;
    const int rc = fla_cycle_scan(x, delta, A, Bm, Cm, y, ws, nws, B, L, d, N, r, nullptr);
    if (rc != 0) {
        std::fprintf(stderr, "cycle scan: %s\n", fla_status_string(rc));
        return 1;
    }
    dump(dir, "x", x, nx);
    dump(dir, "delta", delta, nx);
    dump(dir, "A", A, na);
    dump(dir, "Bm", Bm, nb);
    dump(dir, "Cm", Cm, nb);
    dump(dir, "y", y, nx);
    std::printf("ok\n");
    return 0;
}

static void dump_u16(const char* dir, const char* name, const uint16_t* p, size_t n) {
    char path[1024];
    std::snprintf(path, sizeof path, "%s/%s.bf16", dir, name);
    FILE* f = std::fopen(path, "wb");
    std::fwrite(p, 2, n, f);
    std::fclose(f);
}

static std::mt19937& g_rng() {
    static std::mt19937 r(2468);
    return r;
}

static uint16_t* alloc_bf16(size_t n, std::mt19937& g, bool random) {
    uint16_t* p = static_cast<uint16_t*>(std::aligned_alloc(16, ((n * 2 + 15) / 16) * 16));
    std::normal_distribution<float> d(0.f, 1.f);
    for (size_t i = 0; i < n; ++i) {
        const __bf16 x = random ? (__bf16)d(g) : (__bf16)NAN;
        std::memcpy(p + i, &x, 2);
    }
    return p;
}

// The bf16 forward through the C ABI (its matrix-core kernel on the wave-level emulation):
//   run bf16 KIND B heads GRIDS window shift pad_mode head_dim theta scale outdir
// KIND plain, rope or ms; GRIDS "HxW", or "HxW,HxW,..." for ms.  Writes q, k, v, out (.bf16).
static int run_bf16(int argc, char** argv) {
    if (argc != 13) {
        std::fprintf(stderr, "usage: run bf16 KIND B heads GRIDS window shift pad_mode head_dim theta scale outdir\n");
        return 2;
    }
    const char* kind = argv[2];
    const int B = std::atoi(argv[3]), heads = std::atoi(argv[4]);
    int hw[16], ng = 0;
    for (const char* p = argv[5]; *p && ng < 8;) {
        char* e;
        hw[2 * ng] = (int)std::strtol(p, &e, 10);
        hw[2 * ng + 1] = (int)std::strtol(e + 1, &e, 10);
        ++ng;
        p = *e ? e + 1 : e;
    }
    const int k = std::atoi(argv[6]), s = std::atoi(argv[7]), pm = std::atoi(argv[8]), hd = std::atoi(argv[9]);
    const float theta = (float)std::atof(argv[10]), scale = (float)std::atof(argv[11]);
    const char* dir = argv[12];
    size_t L = 0;
    for (int i = 0; i < ng; ++i) L += (size_t)hw[2 * i] * hw[2 * i + 1];
    const size_t rows = L + (pm ? 1 : 0), tok = (size_t)heads * hd;
    std::mt19937 g(4321);
    uint16_t* q = alloc_bf16(B * L * tok, g, true);
    uint16_t* kk = alloc_bf16(B * rows * tok, g, true);
    uint16_t* v = alloc_bf16(B * rows * tok, g, true);
    uint16_t* out = alloc_bf16(B * L * tok, g, false);
    emu_kernel_args = 0;
    int rc;
    if (std::strcmp(kind, "plain") == 0)
        rc = fla_swin_attn_fwd(q, kk, v, out, B, heads, hw[0], hw[1], hd, k, s, pm, nullptr);
    else if (std::strcmp(kind, "rope") == 0)
        rc = fla_swin_attn_rope_fwd(q, kk, v, out, B, heads, hw[0], hw[1], hd, k, s, pm, theta, scale, nullptr);
    else
        rc = fla_swin_attn_ms_fwd(q, kk, v, out, B, heads, ng, hw, hd, k, s, pm, nullptr);
    if (rc != 0) {
        std::fprintf(stderr, "bf16 forward: %s\n", fla_status_string(rc));
        return 1;
    }
    dump_u16(dir, "q", q, B * L * tok);
    dump_u16(dir, "k", kk, B * rows * tok);
    dump_u16(dir, "v", v, B * rows * tok);
    dump_u16(dir, "out", out, B * L * tok);
    for (uint16_t* p : {q, kk, v, out}) std::free(p);
    std::printf("ok\n");
    return 0;
}

// bf16 training (forward keeping the log-sum-exp, then the backward) through the C ABI:
//   run bf16train KIND B heads GRIDS window shift pad_mode theta scale outdir
// KIND plain, rope or ms; GRIDS as for bf16.  Writes q, k, v, dout, out, dq, dk, dv (.bf16) and
// lse (.f32).
static int run_bf16_train(int argc, char** argv) {
    if (argc != 12) {
        std::fprintf(stderr, "usage: run bf16train KIND B heads GRIDS window shift pad_mode theta scale outdir\n");
        return 2;
    }
    const char* kind = argv[2];
    const int B = std::atoi(argv[3]), heads = std::atoi(argv[4]);
    int hw[16], ng = 0;
    for (const char* p = argv[5]; *p && ng < 8;) {
        char* e;
        hw[2 * ng] = (int)std::strtol(p, &e, 10);
        hw[2 * ng + 1] = (int)std::strtol(e + 1, &e, 10);
        ++ng;
        p = *e ? e + 1 : e;
    }
    const int k = std::atoi(argv[6]), s = std::atoi(argv[7]), pm = std::atoi(argv[8]);
    const float theta = (float)std::atof(argv[9]), scale = (float)std::atof(argv[10]);
    const char* dir = argv[11];
    const int hd = 64;
    size_t L = 0;
    for (int i = 0; i < ng; ++i) L += (size_t)hw[2 * i] * hw[2 * i + 1];
    const size_t rows = L + (pm ? 1 : 0), tok = (size_t)heads * hd;
    std::mt19937 g(8765);
    uint16_t* q = alloc_bf16(B * L * tok, g, true);
    uint16_t* kk = alloc_bf16(B * rows * tok, g, true);
    uint16_t* v = alloc_bf16(B * rows * tok, g, true);
    uint16_t* dout = alloc_bf16(B * L * tok, g, true);
    uint16_t* out = alloc_bf16(B * L * tok, g, false);
    uint16_t* dq = alloc_bf16(B * L * tok, g, false);
    uint16_t* dk = alloc_bf16(B * rows * tok, g, false);
    uint16_t* dv = alloc_bf16(B * rows * tok, g, false);
    float* lse = static_cast<float*>(std::aligned_alloc(16, (((size_t)B * heads * L * 4 + 15) / 16) * 16));
    size_t nws = 0;
    if (fla_swin_attn_bwd_workspace(B, heads, ng, hw, k, s, pm, &nws) != 0) return 1;
    void* ws = nws ? std::aligned_alloc(16, ((nws + 15) / 16) * 16) : nullptr;
    const bool rope = std::strcmp(kind, "rope") == 0, ms = std::strcmp(kind, "ms") == 0;
    emu_kernel_args = 0;
    int rc = rope ? fla_swin_attn_rope_fwd_lse(q, kk, v, out, lse, B, heads, hw[0], hw[1], hd, k, s, pm, theta, scale,
                                               nullptr)
             : ms ? fla_swin_attn_ms_fwd_lse(q, kk, v, out, lse, B, heads, ng, hw, hd, k, s, pm, nullptr)
                  : fla_swin_attn_fwd_lse(q, kk, v, out, lse, B, heads, hw[0], hw[1], hd, k, s, pm, nullptr);
    if (rc != 0) {
        std::fprintf(stderr, "bf16 training forward: %s\n", fla_status_string(rc));
        return 1;
    }
    emu_kernel_args = 1;
    rc = rope ? fla_swin_attn_rope_bwd(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, hw[0], hw[1], hd, k, s,
                                       pm, theta, scale, nullptr)
         : ms ? fla_swin_attn_ms_bwd(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, ng, hw, hd, k, s, pm,
                                     nullptr)
              : fla_swin_attn_bwd(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, hw[0], hw[1], hd, k, s, pm,
                                  nullptr);
    if (rc != 0) {
        std::fprintf(stderr, "bf16 backward: %s\n", fla_status_string(rc));
        return 1;
    }
    if (std::strcmp(kind, "plain") == 0) {
        // the allocation-free backward (its workspace in the library's static array) gives the
        // same bits, twice in a row
        uint16_t* g[3] = {alloc_bf16(B * L * tok, g_rng(), false), alloc_bf16(B * rows * tok, g_rng(), false),
                          alloc_bf16(B * rows * tok, g_rng(), false)};
        const uint16_t* want[3] = {dq, dk, dv};
        const size_t n[3] = {B * L * tok, B * rows * tok, B * rows * tok};
        for (int rep = 0; rep < 2; ++rep) {
            rc = fla_swin_attn_bwd_noalloc(q, kk, v, out, dout, lse, g[0], g[1], g[2], B, heads, hw[0], hw[1], hd, k,
                                           s, pm, nullptr);
            if (rc != 0) {
                std::fprintf(stderr, "allocation-free backward: %s\n", fla_status_string(rc));
                return 1;
            }
            for (int i = 0; i < 3; ++i)
                if (std::memcmp(g[i], want[i], n[i] * 2) != 0) {
                    std::fprintf(stderr, "allocation-free backward differs (gradient %d, call %d)\n", i, rep);
                    return 1;
                }
        }
        for (uint16_t* p : g) std::free(p);
    }
    dump_u16(dir, "q", q, B * L * tok);
    dump_u16(dir, "k", kk, B * rows * tok);
    dump_u16(dir, "v", v, B * rows * tok);
    dump_u16(dir, "dout", dout, B * L * tok);
    dump_u16(dir, "out", out, B * L * tok);
    dump_u16(dir, "dq", dq, B * L * tok);
    dump_u16(dir, "dk", dk, B * rows * tok);
    dump_u16(dir, "dv", dv, B * rows * tok);
    dump(dir, "lse", lse, (size_t)B * heads * L);
    for (uint16_t* p : {q, kk, v, dout, out, dq, dk, dv}) std::free(p);
    std::free(lse);
    std::free(ws);
    std::printf("ok\n");
    return 0;
}

// Launch failure: every entry point must return FLA_ERR_LAUNCH and leave its outputs as they
// were: the emulated runtime is told to fail every launch (the bf16 backward launchers of this
// build, which does not contain those kernels, fail anyway).
static int run_launchfail() {
    const int B = 1, heads = 2, H = 20, W = 13, k = 8, s = 3;
    const size_t L = (size_t)H * W, rows = L + 1, tok = (size_t)heads * 64;
    const int hw[2] = {H, W};
    std::mt19937 g(99);
    int bad = 0;
    auto expect = [&](const char* what, int rc, const float* buf, const float* copy, size_t n) {
        if (rc != FLA_ERR_LAUNCH) {
            std::fprintf(stderr, "%s: status %d (%s), expected FLA_ERR_LAUNCH\n", what, rc, fla_status_string(rc));
            ++bad;
        }
        if (std::memcmp(buf, copy, n * 4) != 0) {
            std::fprintf(stderr, "%s: output changed\n", what);
            ++bad;
        }
    };
    for (int f32 = 0; f32 < 2; ++f32) {
        emu_fail_launch = 1;
        // fp32 sizes throughout: a bf16 call reads and writes half as many bytes
        float* q = alloc_random(B * L * tok, g);
        float* kk = alloc_random(B * rows * tok, g);
        float* v = alloc_random(B * rows * tok, g);
        float* dout = alloc_random(B * L * tok, g);
        float* lse = alloc_random((size_t)B * heads * L, g);
        float* out = alloc_random(B * L * tok, g);
        float* dq = alloc_random(B * L * tok, g);
        float* dk = alloc_random(B * rows * tok, g);
        float* dv = alloc_random(B * rows * tok, g);
        float* keep = alloc_random(B * rows * tok, g);
        size_t nws = 0;
        if (fla_swin_attn_bwd_workspace(B, heads, 1, hw, k, s, 1, &nws) != 0) return 1;
        float* ws = alloc_random(nws / 4 + 1, g);
        float* ws_copy = alloc_random(nws / 4 + 1, g);
        std::memcpy(ws_copy, ws, nws);
        for (int pm = 0; pm < 2; ++pm) {
            std::memcpy(keep, out, B * L * tok * 4);
            emu_kernel_args = 0;
            const int rc = f32 ? fla_swin_attn_fwd_f32(q, kk, v, out, B, heads, H, W, 64, k, s, pm, nullptr)
                               : fla_swin_attn_fwd(q, kk, v, out, B, heads, H, W, 64, k, s, pm, nullptr);
            expect(f32 ? "forward fp32" : "forward bf16", rc, out, keep, B * L * tok);
            std::memcpy(keep, lse, (size_t)B * heads * L * 4);
            const int rl = f32 ? fla_swin_attn_fwd_lse_f32(q, kk, v, out, lse, B, heads, H, W, 64, k, s, pm, nullptr)
                               : fla_swin_attn_fwd_lse(q, kk, v, out, lse, B, heads, H, W, 64, k, s, pm, nullptr);
            expect(f32 ? "training forward fp32 (lse)" : "training forward bf16 (lse)", rl, lse, keep,
                   (size_t)B * heads * L);
            float* grads[3] = {dq, dk, dv};
            const size_t sizes[3] = {B * L * tok, B * rows * tok, B * rows * tok};
            float* copies[3];
            for (int i = 0; i < 3; ++i) {
                copies[i] = alloc_random(sizes[i], g);
                std::memcpy(copies[i], grads[i], sizes[i] * 4);
            }
            emu_kernel_args = 1;
            const int rb = f32 ? fla_swin_attn_bwd_f32(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, H, W,
                                                       64, k, s, pm, nullptr)
                               : fla_swin_attn_bwd(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, H, W, 64,
                                                   k, s, pm, nullptr);
            const char* names[3] = {"backward dq", "backward dk", "backward dv"};
            for (int i = 0; i < 3; ++i) {
                expect(names[i], rb, grads[i], copies[i], sizes[i]);
                std::free(copies[i]);
            }
            expect("backward workspace", rb, ws, ws_copy, nws / 4);
        }
        for (float* p : {q, kk, v, dout, lse, out, dq, dk, dv, keep, ws, ws_copy}) std::free(p);
    }
    // Cycle-scan (fp32 kernels of this build): the runtime fails the launch
    emu_fail_launch = 1;
    emu_kernel_args = 2;
    {
        const int Bc = 1, Lc = 40, d = 10, N = 4;
        float* x = alloc_random((size_t)Bc * Lc * d, g);
        float* dl = alloc_random((size_t)Bc * Lc * d, g);
        float* A = alloc_random((size_t)d * N, g);
        float* Bm = alloc_random((size_t)Bc * Lc * N, g);
        float* Cm = alloc_random((size_t)Bc * Lc * N, g);
        float* y = alloc_random((size_t)Bc * Lc * d, g);
        float* y_copy = alloc_random((size_t)Bc * Lc * d, g);
        std::memcpy(y_copy, y, (size_t)Bc * Lc * d * 4);
        size_t nws = 0;
        if (fla_cycle_scan_workspace(Bc, Lc, d, N, 3, &nws) != 0) return 1;
        void* ws = std::aligned_alloc(16, ((nws + 15) / 16) * 16);
        const int rc = fla_cycle_scan(x, dl, A, Bm, Cm, y, ws, nws, Bc, Lc, d, N, 3, nullptr);
        expect("cycle scan", rc, y, y_copy, (size_t)Bc * Lc * d);
        for (float* p : {x, dl, A, Bm, Cm, y, y_copy}) std::free(p);
        std::free(ws);
    }
    emu_fail_launch = 0;
    if (bad) return 1;
    std::printf("ok\n");
    return 0;
}

int main(int argc, char** argv) {
    if (argc > 1 && std::strcmp(argv[1], "cycle") == 0) return run_cycle(argc, argv);
    if (argc > 1 && std::strcmp(argv[1], "launchfail") == 0) return run_launchfail();
    if (argc > 1 && std::strcmp(argv[1], "bf16") == 0) return run_bf16(argc, argv);
    if (argc > 1 && std::strcmp(argv[1], "bf16train") == 0) return run_bf16_train(argc, argv);
    if (argc != 9) {
        std::fprintf(stderr, "usage: run B heads H W window shift pad_mode outdir\n");
        return 2;
    }
    const int B = std::atoi(argv[1]), heads = std::atoi(argv[2]), H = std::atoi(argv[3]), W = std::atoi(argv[4]);
    const int k = std::atoi(argv[5]), s = std::atoi(argv[6]), pm = std::atoi(argv[7]);
    const char* dir = argv[8];
    const size_t L = (size_t)H * W, rows = L + (pm ? 1 : 0), tok = (size_t)heads * 64;
    std::mt19937 g(1234);
    float* q = alloc_random(B * L * tok, g);
    float* kk = alloc_random(B * rows * tok, g);
    float* v = alloc_random(B * rows * tok, g);
    float* dout = alloc_random(B * L * tok, g);
    float* out = alloc_random(B * L * tok, g);
    float* lse = alloc_random((size_t)B * heads * L, g);
    float* dq = alloc_random(B * L * tok, g);
    float* dk = alloc_random(B * rows * tok, g);
    float* dv = alloc_random(B * rows * tok, g);
    const int hw[2] = {H, W};
    size_t nws = 0;
    if (fla_swin_attn_bwd_workspace(B, heads, 1, hw, k, s, pm, &nws) != 0) return 1;
    void* ws = nws ? std::aligned_alloc(16, ((nws + 15) / 16) * 16) : nullptr;
    emu_kernel_args = 0;
    int rc = fla_swin_attn_fwd_lse_f32(q, kk, v, out, lse, B, heads, H, W, 64, k, s, pm, nullptr);
    if (rc != 0) {
        std::fprintf(stderr, "forward: %s\n", fla_status_string(rc));
        return 1;
    }
    emu_kernel_args = 1;
    rc = fla_swin_attn_bwd_f32(q, kk, v, out, dout, lse, dq, dk, dv, ws, nws, B, heads, H, W, 64, k, s, pm, nullptr);
    if (rc != 0) {
        std::fprintf(stderr, "backward: %s\n", fla_status_string(rc));
        return 1;
    }
    dump(dir, "q", q, B * L * tok);
    dump(dir, "k", kk, B * rows * tok);
    dump(dir, "v", v, B * rows * tok);
    dump(dir, "dout", dout, B * L * tok);
    dump(dir, "out", out, B * L * tok);
    dump(dir, "lse", lse, (size_t)B * heads * L);
    dump(dir, "dq", dq, B * L * tok);
    dump(dir, "dk", dk, B * rows * tok);
    dump(dir, "dv", dv, B * rows * tok);
    std::printf("ok\n");
    return 0;
}
