// Device-side helpers shared by the CAP kernels (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cap.h"

namespace cap {

constexpr int kWave = 64;
constexpr int kMaxK = 8;
constexpr int kMaxE = 256;
constexpr int kMaxR = 64;
constexpr int kMaxDevices = 64;                       // per-device caches of host code
constexpr size_t kLayoutScratchBytes = size_t(4) << 20;   // cap_dispatch_layout_static's workspace

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
// 16-byte raw vector (native clang vector: stays in registers, unlike HIP's uint4 struct)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// bf16 <-> fp32 on raw 16-bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// Two fp32 -> packed bf16x2 (low half = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
}

// Two fp32 -> packed bf16x2 with the hardware conversion (v_cvt_pk_bf16_f32,
// round to nearest even: the same bits as pack_bf16x2 for finite inputs).
typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2_rne(float a, float b) {
    const bf16x2_hw v = {static_cast<__bf16>(a), static_cast<__bf16>(b)};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Mask of lanes below the calling lane.
__device__ __forceinline__ uint64_t lanemask_lt() {
    const int l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// floor(n / d) for 0 <= n < 2^31 and 1 <= d < 2^31 with a quotient below
// 2^16: the fp32 estimate n * rcp(d) is within 2^-21 of n / d relative (so
// within one of the quotient), and one correction step each way makes it exact.
__device__ __forceinline__ int small_quotient(int n, int d) {
    int q = static_cast<int>(static_cast<float>(n) * __builtin_amdgcn_rcpf(static_cast<float>(d)));
    const long long r = static_cast<long long>(n) - static_cast<long long>(q) * d;
    q += (r >= d) ? 1 : 0;
    q -= (r < 0) ? 1 : 0;
    return q;
}

// Grid-wide launch helpers: compute units and XCDs of the current device.
int device_cu_count();
int device_xcc_count();

}  // namespace cap

#define CAP_LAUNCH_CHECK()                                      \
    do {                                                        \
        if (hipGetLastError() != hipSuccess) return CAP_ERR_HIP; \
    } while (0)
