// Host definitions of the gfx950 builtins the kernels use, so that their unmodified sources
// (and the unmodified device header) build as ordinary C++ for the CPU launch emulation
// (test infrastructure; force-included into every file of the host build).
//
// Lane-local builtins are plain functions.  The wave-level ones (the 32x32x16 bf16 matrix
// product, the half-wave swap, the ballot) exchange their operands through a per-wave slot
// area between two barriers over the wave's 64 lanes, which the launch emulation provides:
// every lane of a wave must reach them together, as on the hardware, or the run deadlocks
// (the tests bound it with a time limit).  Buffer resources keep the base and the byte
// range; a load outside the range returns zeros and a store outside it is dropped, dword by
// dword, as the hardware's range check does, and everything inside the range is a real access
// of the caller's allocation (AddressSanitizer sees it).
#pragma once
#include <cmath>
#include <cstdint>
#include <cstring>
#include <type_traits>

#define amdgpu_waves_per_eu(...)

typedef __bf16 emu_bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 emu_bf16x2 __attribute__((ext_vector_type(2)));
typedef float emu_floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned emu_u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned emu_u32x2 __attribute__((ext_vector_type(2)));

// provided by the launch emulation (emu.cpp)
unsigned emu_lane_id();
void emu_wave_barrier();
unsigned char* emu_wave_slots();   // this wave's 64 slots of 64 bytes

inline unsigned __float_as_uint(float x) {
    unsigned u;
    std::memcpy(&u, &x, 4);
    return u;
}
inline float __uint_as_float(unsigned u) {
    float x;
    std::memcpy(&x, &u, 4);
    return x;
}
inline unsigned __umulhi(unsigned a, unsigned b) { return (unsigned)(((unsigned long long)a * b) >> 32); }

inline float __builtin_amdgcn_exp2f(float x) { return std::exp2(x); }
// the hardware sine and cosine take the angle in revolutions
inline float __builtin_amdgcn_cosf(float t) { return (float)std::cos(6.283185307179586 * (double)t); }
inline float __builtin_amdgcn_sinf(float t) { return (float)std::sin(6.283185307179586 * (double)t); }
inline float __builtin_amdgcn_fdot2_f32_bf16(emu_bf16x2 a, emu_bf16x2 b, float c, bool) {
    return (float)a[0] * (float)b[0] + (float)a[1] * (float)b[1] + c;
}

struct __amdgpu_buffer_rsrc_t {
    unsigned char* base;
    unsigned bytes;
};
inline __amdgpu_buffer_rsrc_t __builtin_amdgcn_make_buffer_rsrc(void* p, short, int bytes, int) {
    return __amdgpu_buffer_rsrc_t{static_cast<unsigned char*>(p), (unsigned)bytes};
}
inline emu_u32x4 __builtin_amdgcn_raw_buffer_load_b128(__amdgpu_buffer_rsrc_t r, unsigned off, int soff, int) {
    emu_u32x4 v = {0u, 0u, 0u, 0u};
    const unsigned long long o = (unsigned long long)off + (unsigned)soff;
    for (int d = 0; d < 4; ++d)
        if (o + 4 * d + 4 <= r.bytes) {
            unsigned w;
            std::memcpy(&w, r.base + o + 4 * d, 4);
            v[d] = w;
        }
    return v;
}
inline unsigned __builtin_amdgcn_raw_buffer_load_b32(__amdgpu_buffer_rsrc_t r, unsigned off, int soff, int) {
    const unsigned long long o = (unsigned long long)off + (unsigned)soff;
    unsigned w = 0;
    if (o + 4 <= r.bytes) std::memcpy(&w, r.base + o, 4);
    return w;
}
inline void __builtin_amdgcn_raw_buffer_store_b128(emu_u32x4 v, __amdgpu_buffer_rsrc_t r, unsigned off, int soff,
                                                   int) {
    const unsigned long long o = (unsigned long long)off + (unsigned)soff;
    for (int d = 0; d < 4; ++d)
        if (o + 4 * d + 4 <= r.bytes) {
            const unsigned w = v[d];
            std::memcpy(r.base + o + 4 * d, &w, 4);
        }
}

// D = A B + C, A 32 x 16, B 16 x 32, fp32 accumulation.  Lane l supplies row l % 32 of A and
// column l % 32 of B, elements 8 (l / 32) .. + 7 of the reduction; it receives column l % 32
// of D, rows 8 (r / 4) + 4 (l / 32) + r % 4 for r = 0 .. 15.
inline emu_floatx16 __builtin_amdgcn_mfma_f32_32x32x16_bf16(emu_bf16x8 a, emu_bf16x8 b, emu_floatx16 c, int, int,
                                                           int) {
    struct Slot {
        emu_bf16x8 a, b;
    };
    static_assert(sizeof(Slot) <= 64, "slot");
    Slot* s = reinterpret_cast<Slot*>(emu_wave_slots());
    const unsigned l = emu_lane_id();
    s[l].a = a;
    s[l].b = b;
    emu_wave_barrier();
    const unsigned n = l & 31, h = l >> 5;
    emu_floatx16 d = c;
    for (int r = 0; r < 16; ++r) {
        const unsigned i = 8 * (r >> 2) + 4 * h + (r & 3);
        float acc = 0.f;
        for (int k = 0; k < 16; ++k)
            acc += (float)s[i + 32 * (k >> 3)].a[k & 7] * (float)s[n + 32 * (k >> 3)].b[k & 7];
        d[r] += acc;
    }
    emu_wave_barrier();
    return d;
}

// Swaps the upper 32 lanes of the first operand with the lower 32 lanes of the second:
// returns (new first, new second).
inline emu_u32x2 __builtin_amdgcn_permlane32_swap(unsigned x, unsigned y, bool, bool) {
    unsigned* s = reinterpret_cast<unsigned*>(emu_wave_slots());
    const unsigned l = emu_lane_id();
    s[2 * l] = x;
    s[2 * l + 1] = y;
    emu_wave_barrier();
    emu_u32x2 r;
    if (l < 32) {
        r[0] = x;
        r[1] = s[2 * (l + 32)];
    } else {
        r[0] = s[2 * (l - 32) + 1];
        r[1] = y;
    }
    emu_wave_barrier();
    return r;
}

inline unsigned long long __builtin_amdgcn_ballot_w64(bool p) {
    unsigned char* s = emu_wave_slots();
    const unsigned l = emu_lane_id();
    s[l] = p ? 1 : 0;
    emu_wave_barrier();
    unsigned long long m = 0;
    for (int i = 0; i < 64; ++i)
        if (s[i]) m |= 1ull << i;
    emu_wave_barrier();
    return m;
}

// ---- used by the bf16 backward kernels

typedef short emu_shortx4 __attribute__((ext_vector_type(4)));

// Transposing LDS read: lane i of each 16-lane group names a 4-element piece (row i / 4,
// elements 4 (i % 4) .. + 3) of a 4 x 16 block of 16-bit elements and receives the block's
// column i.
inline emu_shortx4 __builtin_amdgcn_ds_read_tr16_b64_v4i16(__attribute__((address_space(3))) emu_shortx4* p) {
    emu_shortx4* s = reinterpret_cast<emu_shortx4*>(emu_wave_slots());
    const unsigned l = emu_lane_id();
    emu_shortx4 mine;
    std::memcpy(&mine, (const void*)(uintptr_t)p, 8);
    s[l] = mine;
    emu_wave_barrier();
    const unsigned g = l & ~15u, i = l & 15u;
    emu_shortx4 r;
    for (int row = 0; row < 4; ++row) r[row] = s[g + 4 * row + i / 4][i % 4];
    emu_wave_barrier();
    return r;
}

// A buffer load that writes LDS: lane l's `size` bytes go to the LDS address base + l * size
// (zeros outside the buffer's range), here at once.  The wave's wait for its loads is where the
// rows its lanes wrote become visible to the whole wave: a barrier over the wave's lanes.
inline void __builtin_amdgcn_raw_ptr_buffer_load_lds(__amdgpu_buffer_rsrc_t r, __attribute__((address_space(3))) void* lds,
                                                    unsigned size, unsigned voff, unsigned soff, unsigned off,
                                                    unsigned) {
    unsigned char* dst = (unsigned char*)(uintptr_t)lds + (size_t)emu_lane_id() * size;
    const unsigned long long o = (unsigned long long)voff + soff + off;
    for (unsigned d = 0; d < size; d += 4) {
        unsigned w = 0;
        if (o + d + 4 <= r.bytes) std::memcpy(&w, r.base + o + d, 4);
        std::memcpy(dst + d, &w, 4);
    }
}
inline void __builtin_amdgcn_s_waitcnt(int) { emu_wave_barrier(); }

inline int __builtin_amdgcn_readfirstlane(int x) {
    int* s = reinterpret_cast<int*>(emu_wave_slots());
    s[emu_lane_id()] = x;
    emu_wave_barrier();
    const int r = s[0];
    emu_wave_barrier();
    return r;
}

template <typename T>
inline T __shfl_xor(T x, int mask, int = 64) {
    static_assert(sizeof(T) == 4, "32-bit shuffles");
    T* s = reinterpret_cast<T*>(emu_wave_slots());
    const unsigned l = emu_lane_id();
    s[l] = x;
    emu_wave_barrier();
    const T r = s[(l ^ (unsigned)mask) & 63u];
    emu_wave_barrier();
    return r;
}
