// Host-side bounds checker of the library's kernels (test infrastructure).
//
// This program is linked from the library's own sources compiled for the CPU
// only (no device code), with AddressSanitizer and UndefinedBehaviorSanitizer
// on all host code, and installs a launch observer: the C ABI entry points run
// their argument checks, sign table and kernel choice exactly as in the GPU
// library, and every launch's plan (kernel, template arguments, grid, LDS
// bytes, argument block) comes to this program instead of a GPU.  The device
// pointers are fake addresses that are never dereferenced; each names a
// buffer of known size.  For every plan the checker walks the kernel's
// address arithmetic -- the functions the kernel itself calls -- over every
// workgroup and lane (see check_conv_mfma.cpp and friends) and reports any
// access outside its buffer, any LDS word read that the stage did not write
// or that holds another element than the one the product needs, and any
// output written twice or never.
//
// Input: one case per line on stdin,
//   conv   k g_1..g_k B C_in C_out d_image d_filter algo  ACT
//   block  k g_1..g_k B C_in C_mid C_out d_image d_filter path  ACT ACT
//   act    nb B C P  ACT
//   fastdiv  (the reciprocal division of the kernels' index arithmetic)
// with ACT = mode K blade_1..blade_K (mode -1: none, K then 0).
// Output: one line per case, "ok <status> <launches> <simulated workgroups>
// <kernel kinds> <tiles>" (kinds: the LaunchKind of each launch,
// comma-separated, or "-"; tiles: each launch's template arguments joined by
// '.', comma-separated, or "-") or "FAIL <message>".
#include <inttypes.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <sstream>
#include <string>
#include <vector>

#include "check.hpp"
#include "cliffconv.h"
#include "conv_mfma_geom.hpp"

namespace hostcheck {

Case* current = nullptr;

void fail(const char* fmt, ...)
{
    if (current->errors++ < 8) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        if (!current->first_error.empty()) current->first_error += " | ";
        current->first_error += buf;
    }
}

const Buffer* find_buffer(const void* p)
{
    for (const Buffer& b : current->buffers)
        if (b.ptr == p) return &b;
    return nullptr;
}

// Fake device address space: buffers are laid out from 2^44 on, 4 KiB
// apart and 256-byte aligned; nothing ever dereferences them.
static uintptr_t next_addr;

static float* make_buffer(const char* name, int64_t n_floats)
{
    if (n_floats <= 0) return nullptr;
    Buffer b;
    b.name = name;
    float* p = reinterpret_cast<float*>(next_addr);
    b.ptr = p;
    b.n = n_floats;
    current->buffers.push_back(b);
    next_addr += ((uintptr_t)n_floats * 4 + 4096 + 255) & ~(uintptr_t)255;
    return p;
}

static void on_launch(const cliff::LaunchPlan& p, void*)
{
    current->launches++;
    if (!current->kinds.empty()) current->kinds += ",";
    current->kinds += std::to_string(p.kind);
    if (!current->tiles.empty()) current->tiles += ",";
    for (int t = 0; t < 12; ++t) current->tiles += (t ? "." : "") + std::to_string(p.tpl[t]);
    switch (p.kind) {
    case cliff::LAUNCH_CONV_MFMA: check_conv_mfma(p); break;
    case cliff::LAUNCH_CONV1D_MFMA: check_conv1d(p); break;
    case cliff::LAUNCH_BLOCK_SMALL: check_block_small(p); break;
    case cliff::LAUNCH_ACT: check_act(p); break;
    case cliff::LAUNCH_LINEAR_MFMA: check_linear(p); break;
    case cliff::LAUNCH_CONV_DIRECT: check_direct(p); break;
    default: check_generic(p); break;
    }
}

}  // namespace hostcheck

using namespace hostcheck;

static int64_t ipow(int64_t a, int k)
{
    int64_t r = 1;
    for (int t = 0; t < k; ++t) r *= a;
    return r;
}

struct Act {
    bool on = false;
    cliff_act_desc d;
};

static bool read_act(std::istringstream& in, Act& a)
{
    int mode, K;
    if (!(in >> mode >> K)) return false;
    memset(&a.d, 0, sizeof a.d);
    a.on = mode >= 0;
    a.d.mode = mode;
    a.d.K = K;
    for (int t = 0; t < K; ++t)
        if (!(in >> a.d.blade_idx[t])) return false;
    return true;
}

static void act_buffers(Act& a, int64_t C, const char* wname, const char* bname)
{
    if (a.on && a.d.mode == CLIFF_AGG_LINEAR) {
        a.d.weight = make_buffer(wname, C * a.d.K);
        a.d.bias = make_buffer(bname, C);
    }
}

int main()
{
    cliff::LaunchObserver obs{256, on_launch, nullptr};
    cliff::launch_observer = &obs;
    std::string line;
    while (std::getline(std::cin, line)) {
        if (line.empty() || line[0] == '#') continue;
        std::istringstream in(line);
        std::string kind;
        in >> kind;
        Case c;
        current = &c;
        next_addr = (uintptr_t)1 << 44;
        int st = -1;
        if (kind == "conv" || kind == "block") {
            int k;
            in >> k;
            int8_t g[3] = {0, 0, 0};
            for (int t = 0; t < k && t < 3; ++t) {
                int v;
                in >> v;
                g[t] = (int8_t)v;
            }
            const int nb = 1 << k;
            if (kind == "conv") {
                int64_t B, C_in, C_out, D, df;
                int algo;
                Act a;
                if (!(in >> B >> C_in >> C_out >> D >> df >> algo) || !read_act(in, a)) {
                    printf("FAIL bad case line\n");
                    continue;
                }
                const int64_t Do = D - df + 1;
                c.dims = {k, nb, B, C_in, C_out, D, df};
                const float* x = make_buffer("input", B * C_in * ipow(D, k) * nb);
                const float* w = make_buffer("filters", C_in * C_out * ipow(df, k) * nb);
                const float* b = make_buffer("bias", C_out * nb);
                act_buffers(a, C_out, "act weight", "act bias");
                float* y = make_buffer("output", B * C_out * ipow(Do, k) * nb);
                if (!x) x = make_buffer("input", 4);
                if (!y) y = make_buffer("output", 4);
                st = clifford_conv_nd_algo(k, g, B, C_in, C_out, D, df, x, w, b, y,
                                           a.on ? &a.d : nullptr, nullptr, algo);
            } else {
                int64_t B, C_in, C_mid, C_out, D, df;
                int path;
                Act a1, a2;
                if (!(in >> B >> C_in >> C_mid >> C_out >> D >> df >> path) || !read_act(in, a1) ||
                    !read_act(in, a2)) {
                    printf("FAIL bad case line\n");
                    continue;
                }
                const int64_t Dm = D - df + 1, Do = Dm - df + 1;
                c.dims = {k, nb, B, C_in, C_out, D, df};
                const float* x = make_buffer("input", B * C_in * ipow(D, k) * nb);
                const float* w1 = make_buffer("filters1", C_in * C_mid * ipow(df, k) * nb);
                const float* b1 = make_buffer("bias1", C_mid * nb);
                const float* w2 = make_buffer("filters2", C_mid * C_out * ipow(df, k) * nb);
                const float* b2 = make_buffer("bias2", C_out * nb);
                act_buffers(a1, C_mid, "act1 weight", "act1 bias");
                act_buffers(a2, C_out, "act2 weight", "act2 bias");
                float* ws = make_buffer("workspace", B * C_mid * ipow(Dm, k) * nb);
                float* y = make_buffer("output", B * C_out * ipow(Do, k) * nb);
                if (!x) x = make_buffer("input", 4);
                if (!ws) ws = make_buffer("workspace", 4);
                if (!y) y = make_buffer("output", 4);
                st = clifford_block2_nd_path(k, g, B, C_in, C_mid, C_out, D, df, x, w1, b1,
                                             a1.on ? &a1.d : nullptr, w2, b2,
                                             a2.on ? &a2.d : nullptr, ws, y, nullptr, path);
            }
        } else if (kind == "fastdiv") {
            // the kernels' division by a reciprocal (conv_mfma_geom.hpp)
            // against integer division: every n below 2^20 for d below 64,
            // random pairs over the whole non-negative int range, and the
            // quotient boundaries q d - 1, q d near the top of the range
            uint64_t rs = 0x9E3779B97F4A7C15ull;
            auto rnd = [&]() {
                rs ^= rs << 13;
                rs ^= rs >> 7;
                rs ^= rs << 17;
                return rs;
            };
            auto check = [&](int n, int d) {
                if (cliff::fdiv(n, cliff::fast_div(d)) != n / d)
                    fail("fdiv %d / %d gives %d", n, d, cliff::fdiv(n, cliff::fast_div(d)));
            };
            for (int d = 1; d < 64 && !c.errors; ++d)
                for (int n = 0; n < (1 << 20); ++n) check(n, d);
            for (int i = 0; i < 4000000 && c.errors < 4; ++i) {
                const int d = 1 + (int)(rnd() % (i & 1 ? 0x7FFFFFFFull : 100000ull));
                const int n = (int)(rnd() & 0x7FFFFFFF);
                check(n, d);
                const int q = (0x7FFFFFFF - (int)(rnd() % 1000)) / d;
                check(q * d, d);
                if (q * d > 0) check(q * d - 1, d);
            }
            st = 0;
        } else if (kind == "act") {
            int nb;
            int64_t B, C, P;
            Act a;
            if (!(in >> nb >> B >> C >> P) || !read_act(in, a)) {
                printf("FAIL bad case line\n");
                continue;
            }
            c.dims = {0, nb, B, C, C, P, 1};
            const float* x = make_buffer("input", B * C * P * nb);
            act_buffers(a, C, "act weight", "act bias");
            float* y = make_buffer("output", B * C * P * nb);
            if (!x) x = make_buffer("input", 4);
            if (!y) y = make_buffer("output", 4);
            st = multivector_act(nb, B, C, P, a.on ? &a.d : nullptr, x, y, nullptr);
        } else {
            printf("FAIL unknown case kind %s\n", kind.c_str());
            continue;
        }
        if (c.errors)
            printf("FAIL status %d, %d errors: %s\n", st, c.errors, c.first_error.c_str());
        else
            printf("ok %d %d %" PRId64 " %s %s\n", st, c.launches, c.workgroups,
                   c.kinds.empty() ? "-" : c.kinds.c_str(),
                   c.tiles.empty() ? "-" : c.tiles.c_str());
        fflush(stdout);
    }
    cliff::launch_observer = nullptr;
    return 0;
}
