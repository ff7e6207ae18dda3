// Opt-in per-kernel timing: when enabled, each tagged launch is bracketed by
// two hipEvents recorded on the launch stream, and its algorithmic work
// (flops and bytes the operation must do, not what the kernel happens to do)
// is accumulated under the tag.
#pragma once

#include "common.hpp"

namespace rat3d {

bool prof_on();
int prof_begin(const char* tag, hipStream_t st);
void prof_end(int slot, hipStream_t st, double alg_flops, double alg_bytes);

struct ProfScope {
    int slot;
    hipStream_t st;
    double flops, bytes;
    ProfScope(const char* tag, hipStream_t s, double f, double b)
        : slot(prof_on() ? prof_begin(tag, s) : -1), st(s), flops(f), bytes(b) {}
    ~ProfScope() {
        if (slot >= 0) prof_end(slot, st, flops, bytes);
    }
};

}  // namespace rat3d
