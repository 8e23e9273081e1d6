// Host-side declarations of the Cycle-scan kernels (fla_cycle_scan.hip), shared with the
// C ABI in fla_swin_api.cpp.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace fla {

// Cycle-scan (fla_cycle_scan.hip): selective scan over the sequence laid out `repeats` times.
struct CycleArgs {
    const float* x;       // [B, L, d]
    const float* delta;   // [B, L, d]
    const float* A;       // [d, N]
    const float* Bm;      // [B, L, N]
    const float* Cm;      // [B, L, N]
    float* y;             // [B, L, d]
    float* ws_h;          // [B, nch, d, N]: chunk end states, then the chunks' starting states
    float* ws_s;          // [B, nch, d]: sum of Delta over each chunk
    int B, L, d, N, repeats;
    int T;                // tokens per chunk
    int nch;              // chunks: ceil(L / T)
    int cgroups;          // groups of 64 channels: ceil(d / 64)
    int seg;              // carry pass: segments of chunks per (batch entry, channel, state), 1 to 8
                          // (set by launch_cycle_scan)
};
bool cycle_states_supported(int N);   // N in {1, 2, 4, 8, 16, 32}
// Tokens per chunk: enough chunks to fill the chip at the sizes of an image layer, at
// least 32 tokens (a power of two from 32 to 256).
inline int cycle_chunk(int L) {
    int T = 32;
    while (T < 256 && (int64_t)T * 64 < L) T *= 2;
    return T;
}
inline int64_t cycle_workspace_floats(int B, int L, int d, int N) {
    const int T = cycle_chunk(L);
    const int64_t nch = (L + T - 1) / T;
    return (int64_t)B * nch * d * (N + 1);
}
hipError_t launch_cycle_scan(const CycleArgs& a, hipStream_t stream);

}  // namespace fla
