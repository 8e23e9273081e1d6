// Host stand-in for the HIP pieces the fp32 kernels and the C ABI use, so that their unmodified
// sources build as ordinary C++ and run on the CPU (test infrastructure).  A kernel launch runs
// its blocks one after another, each with blockDim.x host threads; __shared__ arrays become
// statics (one block is live at a time, so they are that block's shared memory) and
// __syncthreads() is a barrier over the block's threads.
#pragma once
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>

#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __shared__ static
#define __launch_bounds__(...)
using std::max;
using std::min;

struct dim3 {
    unsigned x, y, z;
    dim3(unsigned a = 1, unsigned b = 1, unsigned c = 1) : x(a), y(b), z(c) {}
};
struct emu_index {
    unsigned x, y, z;
};
extern thread_local emu_index threadIdx, blockIdx;
void __syncthreads();

struct alignas(16) float4 {
    float x, y, z, w;
};
inline float4 make_float4(float a, float b, float c, float d) { return float4{a, b, c, d}; }
struct alignas(8) float2 {
    float x, y;
};
inline float2 make_float2(float a, float b) { return float2{a, b}; }
struct alignas(16) uint4 {
    unsigned x, y, z, w;
};
struct alignas(8) uint2 {
    unsigned x, y;
};

typedef int hipError_t;
constexpr hipError_t hipSuccess = 0;
constexpr hipError_t hipErrorInvalidValue = 1;
typedef void* hipStream_t;
struct hipDeviceProp_t {
    char gcnArchName[256];
    int multiProcessorCount;
};
hipError_t hipGetDevice(int* device);
hipError_t hipGetDeviceProperties(hipDeviceProp_t* prop, int device);
hipError_t hipGetLastError();
hipError_t hipLaunchKernel(const void* fn, dim3 grid, dim3 block, void** args, size_t shmem, hipStream_t stream);
