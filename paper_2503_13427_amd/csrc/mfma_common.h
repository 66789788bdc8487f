// Device helpers shared by the chunkwise kernels of the xLSTM 7B head shape (DQK = 256, DV = 512):
// bf16 16x16x32 MFMA with fp32 accumulation, the gfx950 LDS transpose read, buffer resources, DPP
// wave scans and the segment-slot layout.  Everything lives in an anonymous namespace, so each
// translation unit that includes this header has its own copy.
#pragma once

#include "device_common.h"

namespace mlstm {
namespace {

constexpr int kDQK = 256;
constexpr int kDV = 512;
constexpr int kDVT = 128;             // dv columns per workgroup
constexpr int kNTile = kDV / kDVT;    // 4 dv tiles per sequence
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kQScale = 0.0625f;    // 1 / sqrt(256), exact

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4_t mfma16(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

// Two fp32 -> packed bf16 pair, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ float lo_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f32(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS transpose read: 4 bf16 per lane (see the header comment for the lane mapping).
__device__ __forceinline__ u32x2_t tr_read(const uint16_t* p) {
    typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p)));
}
__device__ __forceinline__ u32x4_t cat(u32x2_t a, u32x2_t b) { return u32x4_t{a[0], a[1], b[0], b[1]}; }

// Buffer resources (SGPRs) for one sequence's inputs: loads need one 32-bit VGPR
// offset per staging item plus immediate offsets.  Out-of-range reads return zero.
constexpr int kRsrcWord3 = 0x00020000;

struct SeqRsrc {
    __amdgpu_buffer_rsrc_t q, k, v, ig, fg, h;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0), static_cast<int>(bytes),
                                             kRsrcWord3);
}
__device__ __forceinline__ u32x4_t bload128(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ float bloadf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// Inclusive scans over the 64 lanes of a wave with DPP: shifts inside 16-lane rows,
// then the row_bcast steps carry row totals forward.  Lanes without a source take the
// identity (0 for the sum, -inf for the max).
#define MLSTM_DPP(old, x, ctrl, rmask)                                                                   \
    __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, (old)),                 \
                                                          __builtin_bit_cast(int, (x)), (ctrl), (rmask), 0xf, false))
__device__ __forceinline__ float wave_incl_sum(float x) {
    x += MLSTM_DPP(0.0f, x, 0x111, 0xf);   // row_shr:1
    x += MLSTM_DPP(0.0f, x, 0x112, 0xf);   // row_shr:2
    x += MLSTM_DPP(0.0f, x, 0x114, 0xf);   // row_shr:4
    x += MLSTM_DPP(0.0f, x, 0x118, 0xf);   // row_shr:8
    x += MLSTM_DPP(0.0f, x, 0x142, 0xa);   // row_bcast:15 into rows 1 and 3
    x += MLSTM_DPP(0.0f, x, 0x143, 0xc);   // row_bcast:31 into rows 2 and 3
    return x;
}
__device__ __forceinline__ float wave_incl_max(float x) {
    x = fmaxf(x, MLSTM_DPP(-INFINITY, x, 0x111, 0xf));
    x = fmaxf(x, MLSTM_DPP(-INFINITY, x, 0x112, 0xf));
    x = fmaxf(x, MLSTM_DPP(-INFINITY, x, 0x114, 0xf));
    x = fmaxf(x, MLSTM_DPP(-INFINITY, x, 0x118, 0xf));
    x = fmaxf(x, MLSTM_DPP(-INFINITY, x, 0x142, 0xa));
    x = fmaxf(x, MLSTM_DPP(-INFINITY, x, 0x143, 0xc));
    return x;
}
// Segmented inclusive max: a lane with ``start`` set begins a new segment, so every lane gets the
// maximum over the lanes from the last start at or before it (all lanes before it if none).  Each
// step combines (flag, value) pairs with the associative rule "a later start discards the left".
__device__ __forceinline__ float wave_seg_incl_max(float x, bool start) {
    int f = start ? 1 : 0;
#define MLSTM_SEG_STEP(ctrl, rmask)                                                                        \
    {                                                                                                     \
        const float y = MLSTM_DPP(-INFINITY, x, ctrl, rmask);                                             \
        const int fy = __builtin_amdgcn_update_dpp(0, f, (ctrl), (rmask), 0xf, false);                    \
        x = f ? x : fmaxf(x, y);                                                                          \
        f |= fy;                                                                                          \
    }
    MLSTM_SEG_STEP(0x111, 0xf)
    MLSTM_SEG_STEP(0x112, 0xf)
    MLSTM_SEG_STEP(0x114, 0xf)
    MLSTM_SEG_STEP(0x118, 0xf)
    MLSTM_SEG_STEP(0x142, 0xa)
    MLSTM_SEG_STEP(0x143, 0xc)
#undef MLSTM_SEG_STEP
    return x;
}
#undef MLSTM_DPP
// sum over the four 16-lane rows of a wave, in every lane (gfx950 cross-row lane swaps, no LDS)
__device__ __forceinline__ float sum_rows4(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);   // rows (0, 1) <-> (2, 3)
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const uint32_t w = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(w, w, false, false);   // rows 0 <-> 1, 2 <-> 3
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float lane63(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

// exp and log sigmoid through the hardware exp2 / log2 (v_exp_f32, v_log_f32).
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float flogsig(float x) {
    return fminf(x, 0.0f) - 0.6931471805599453f * __builtin_amdgcn_logf(1.0f + fexp(-fabsf(x)));
}

// XCD-aware block order: the hardware deals consecutive workgroups round-robin to
// the 8 XCDs; renumber so that consecutive work items (the four dv tiles of a
// sequence/segment) run on the same XCD.
__device__ __forceinline__ int work_index() {
    const int nb = gridDim.x, b = blockIdx.x;
    if (nb % 8) return b;
    return (b % 8) * (nb / 8) + b / 8;
}

// workspace slot of (sequence s, local sub-segment j): C [DQK*DV], n [DQK], then m_loc, gsum
// (sum of logsig over the sub-segment), m_in (entry max state, in segment-boundary slots), pad.
// C is stored four rows interleaved: element (d, v) at ((d / 4) DV + v) 4 + d % 4, so the four
// consecutive d one accumulator lane holds for one v are one 16-byte piece
__host__ __device__ constexpr int64_t slot_c4(int d4, int v) { return (static_cast<int64_t>(d4) * kDV + v) * 4; }
constexpr int64_t kSlotFloats = static_cast<int64_t>(kDQK) * kDV + kDQK + 4;

}  // namespace
}  // namespace mlstm
