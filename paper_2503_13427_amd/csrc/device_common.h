// Device helpers shared by the libmlstm kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mlstm {

// Debug builds (-DMLSTM_DEBUG): bounds checks on computed indices that record a violation in a
// flag word of the translation unit (one bit per source file) instead of trapping, so a violated
// check never faults the device.  The host collects and clears the words with mlstm_debug_flags().
// In the default build the checks compile to nothing.
#ifdef MLSTM_DEBUG
namespace {
__device__ unsigned int g_debug_flags;
}  // namespace
#define MLSTM_CHECK(cond, bit)                                           \
    do {                                                                 \
        if (!(cond)) atomicOr(&::mlstm::g_debug_flags, (bit));           \
    } while (0)
// Defines `fn(unsigned int* out)`: ORs this translation unit's flag word into *out and clears it.
#define MLSTM_DEBUG_READER(fn)                                                                              \
    hipError_t fn(unsigned int* out) {                                                                      \
        unsigned int v = 0;                                                                                 \
        hipError_t e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_debug_flags), sizeof(v), 0, hipMemcpyDeviceToHost); \
        if (e != hipSuccess) return e;                                                                      \
        *out |= v;                                                                                          \
        v = 0;                                                                                              \
        return hipMemcpyToSymbol(HIP_SYMBOL(g_debug_flags), &v, sizeof(v), 0, hipMemcpyHostToDevice);       \
    }
#else
#define MLSTM_CHECK(cond, bit) ((void)0)
#endif
// bits of the flag word, one per source file
constexpr unsigned int kDbgChunkMfma = 1u, kDbgChunkF32 = 2u, kDbgStep = 4u, kDbgOutputNorm = 8u,
                       kDbgGatePreact = 16u, kDbgChunkBwd = 32u, kDbgParallelBwd = 64u;

// bf16 is carried as its uint16 bit pattern.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even (the hardware conversion, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

template <typename T> struct io;
template <> struct io<float> {
    static __device__ __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float* p, int64_t i, float x) { p[i] = x; }
};
template <> struct io<bf16_t> {
    static __device__ __forceinline__ float load(const bf16_t* p, int64_t i) { return bf16_to_f32(p[i].bits); }
    static __device__ __forceinline__ void store(bf16_t* p, int64_t i, float x) { p[i].bits = f32_to_bf16(x); }
};

// log(sigmoid(x)) = min(x, 0) - log1p(exp(-|x|)); exact for +-inf, no overflow.
__device__ __forceinline__ float logsigmoid(float x) {
    return fminf(x, 0.0f) - log1pf(expf(-fabsf(x)));
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

}  // namespace mlstm
