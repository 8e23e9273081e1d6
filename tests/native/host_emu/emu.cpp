// The launch emulation behind hip_runtime.h (see there), with the wave-level exchange that the
// matrix-core and cross-lane builtins of amdgcn_host.h use, and a device that reports gfx950.
#include <barrier>
#include <memory>
#include <thread>
#include <vector>

#include "fla_cycle_scan.h"
#include "fla_swin_internal.h"

thread_local emu_index threadIdx, blockIdx;
static std::barrier<>* g_block_barrier = nullptr;
void __syncthreads() { g_block_barrier->arrive_and_wait(); }

// waves of 64 work items: a barrier over each wave's lanes and 4 KB of exchange slots per wave
constexpr unsigned kEmuMaxWaves = 16;   // workgroups of up to 1024 work items
static std::vector<std::unique_ptr<std::barrier<>>> g_wave_barriers;
alignas(64) static unsigned char g_wave_slots[kEmuMaxWaves][4096];
unsigned emu_lane_id() { return threadIdx.x & 63u; }
void emu_wave_barrier() { g_wave_barriers[threadIdx.x >> 6]->arrive_and_wait(); }
unsigned char* emu_wave_slots() { return g_wave_slots[threadIdx.x >> 6]; }

hipError_t hipGetDevice(int* device) {
    *device = 0;
    return hipSuccess;
}
hipError_t hipGetDeviceProperties(hipDeviceProp_t* prop, int) {
    std::strcpy(prop->gcnArchName, "gfx950:sramecc+:xnack-");
    prop->multiProcessorCount = 256;
    return hipSuccess;
}
hipError_t hipGetLastError() { return hipSuccess; }

// every kernel the host build launches takes one argument struct; which one is told by the
// caller (emu_kernel_args) before each API call
int emu_kernel_args = 0;   // 0: SwinArgs, 1: SwinBwdArgs, 2: CycleArgs
// nonzero: every launch fails as a real runtime's would on a bad configuration (the launch-failure
// path of the C ABI)
int emu_fail_launch = 0;

hipError_t hipLaunchKernel(const void* fn, dim3 grid, dim3 block, void** args, size_t, hipStream_t) {
    if (emu_fail_launch) return hipErrorInvalidValue;
    const unsigned nw = (block.x + 63) / 64;
    if (nw > kEmuMaxWaves) return hipErrorInvalidValue;
    std::barrier<> bar((std::ptrdiff_t)block.x);
    g_block_barrier = &bar;
    g_wave_barriers.clear();
    for (unsigned w = 0; w < nw; ++w)
        g_wave_barriers.emplace_back(std::make_unique<std::barrier<>>((std::ptrdiff_t)std::min(64u, block.x - 64 * w)));
    for (unsigned b = 0; b < grid.x; ++b) {
        std::vector<std::thread> threads;
        threads.reserve(block.x);
        for (unsigned t = 0; t < block.x; ++t)
            threads.emplace_back([=]() {
                threadIdx = {t, 0, 0};
                blockIdx = {b, 0, 0};
                if (emu_kernel_args == 0)
                    reinterpret_cast<void (*)(fla::SwinArgs)>(const_cast<void*>(fn))(*static_cast<fla::SwinArgs*>(args[0]));
                else if (emu_kernel_args == 1)
                    reinterpret_cast<void (*)(fla::SwinBwdArgs)>(const_cast<void*>(fn))(
                        *static_cast<fla::SwinBwdArgs*>(args[0]));
                else
                    reinterpret_cast<void (*)(fla::CycleArgs)>(const_cast<void*>(fn))(
                        *static_cast<fla::CycleArgs*>(args[0]));
            });
        for (auto& th : threads) th.join();
    }
    g_block_barrier = nullptr;
    g_wave_barriers.clear();
    return hipSuccess;
}

namespace fla {
// the static device array of the allocation-free backward: a host array of the same size
hipError_t scratch_address(void** ptr) {
    alignas(256) static unsigned char scratch[kScratchBytes];
    *ptr = scratch;
    return hipSuccess;
}
}  // namespace fla
