// Shared declarations of the host-side bounds checker (test infrastructure;
// see check_main.cpp).
#pragma once

#include <stdint.h>

#include <iostream>
#include <string>
#include <vector>

#include "common.hpp"

namespace hostcheck {

struct Buffer {
    std::string name;
    const float* ptr;
    int64_t n;  // floats
};

struct Dims {
    int k = 0, nb = 0;
    int64_t B = 0, C_in = 0, C_out = 0, D = 0, df = 0;
};

struct Case {
    std::vector<Buffer> buffers;
    Dims dims;
    int launches = 0;
    int64_t workgroups = 0;  // workgroups whose LDS image was simulated
    bool grid_sampled = false;  // a grid too large to walk every workgroup
    std::string kinds;          // LaunchKind of each launch, comma-separated
    std::string tiles;          // each launch's template values, '.'-joined, comma-separated
    int errors = 0;
    std::string first_error;
};

extern Case* current;

void fail(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
const Buffer* find_buffer(const void* p);

void check_conv_mfma(const cliff::LaunchPlan& p);
void check_conv1d(const cliff::LaunchPlan& p);
void check_block_small(const cliff::LaunchPlan& p);
void check_act(const cliff::LaunchPlan& p);
void check_linear(const cliff::LaunchPlan& p);
void check_direct(const cliff::LaunchPlan& p);
void check_generic(const cliff::LaunchPlan& p);

}  // namespace hostcheck
