// Hidden-state output of the mLSTM cell (Sec. 2, Eq. 6 with the output gate of Eq. 9):
//   h = sigmoid(o~) * (Norm(h~) * weight[head] + bias[head]),
// Norm the headwise LayerNorm or RMSNorm over the DV values of one (batch, head, step) row.
//
// HBM-bound: a row is read once (h~ and o~) and written once.  One wave owns one row and holds
// it in registers (eight contiguous elements per lane and slab), so the mean and the mean squared
// deviation come from two wave reductions over values already loaded, with no second pass over
// memory.
#include <type_traits>

#include "device_common.h"
#include "launch.h"

namespace mlstm {
namespace {

constexpr int kNormThreads = 256;                      // four rows per workgroup
constexpr int kNormMaxSlabs = kOutNormMaxDV / 512;          // eight-element slabs per lane at most

// Sum over the 64 lanes of a wave, in every lane: DPP within each 16-lane row (quad swaps, then
// the half-row and row mirrors), then the gfx950 cross-row lane swaps; no LDS.
#define MLSTM_DPP_ADD(x, ctrl) \
    ((x) + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, (x)), (ctrl), 0xf, 0xf, false)))
__device__ __forceinline__ float wave_total(float x) {
    x = MLSTM_DPP_ADD(x, 0xB1);    // quad_perm [1, 0, 3, 2]
    x = MLSTM_DPP_ADD(x, 0x4E);    // quad_perm [2, 3, 0, 1]
    x = MLSTM_DPP_ADD(x, 0x141);   // row_half_mirror
    x = MLSTM_DPP_ADD(x, 0x140);   // row_mirror
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);   // rows (0, 1) <-> (2, 3)
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const uint32_t v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);   // rows 0 <-> 1, 2 <-> 3
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
#undef MLSTM_DPP_ADD

__device__ __forceinline__ void load4(const float* p, float (&x)[4]) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
}
__device__ __forceinline__ void load4(const bf16_t* p, float (&x)[4]) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    x[0] = __uint_as_float(v.x << 16); x[1] = __uint_as_float(v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.y << 16); x[3] = __uint_as_float(v.y & 0xffff0000u);
}
// eight contiguous elements: one 16-byte access for bf16, two for fp32
__device__ __forceinline__ void load8(const float* p, float* x) {
    load4(p, *reinterpret_cast<float(*)[4]>(x));
    load4(p + 4, *reinterpret_cast<float(*)[4]>(x + 4));
}
__device__ __forceinline__ void load8(const bf16_t* p, float* x) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void store8(float* p, const float* x) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
}
__device__ __forceinline__ void store8(bf16_t* p, const float* x) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        w[i] = static_cast<uint32_t>(f32_to_bf16(x[2 * i])) | (static_cast<uint32_t>(f32_to_bf16(x[2 * i + 1])) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void store4(float* p, const float (&x)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}
__device__ __forceinline__ void store4(bf16_t* p, const float (&x)[4]) {
    uint2 v;
    v.x = static_cast<uint32_t>(f32_to_bf16(x[0])) | (static_cast<uint32_t>(f32_to_bf16(x[1])) << 16);
    v.y = static_cast<uint32_t>(f32_to_bf16(x[2])) | (static_cast<uint32_t>(f32_to_bf16(x[3])) << 16);
    *reinterpret_cast<uint2*>(p) = v;
}

// Lane l holds, in slab j, the eight elements 512 j + 8 l + 0..7 of the row (two four-element
// groups; the second may lie past a row width that is a multiple of 4 but not of 8).  NS slabs
// cover rows up to 512 NS elements, so a narrow row does not pay registers, and occupancy, for the
// widest one.
template <typename TIn, int NS>
__global__ void __launch_bounds__(kNormThreads)
output_norm_kernel(const TIn* ht, const TIn* __restrict__ op, const float* __restrict__ weight,
                   const float* __restrict__ bias, float eps, int rms, int64_t rows, int NH, int T, int DV,
                   TIn* h, RowStrides so, RowStrides sy) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (kNormThreads / 64) + (threadIdx.x >> 6);
    if (row >= rows) return;   // whole waves; the kernel has no barrier
    const int64_t bh = row / T, t = row - bh * T;
    const int64_t bb = bh / NH;
    const int head = static_cast<int>(bh - bb * NH);
    const int ng = DV / 4;
    MLSTM_CHECK(t < T && head < NH && DV % 4 == 0, kDbgOutputNorm);
    const TIn* x = ht + row * DV;
    const TIn* o = op + bb * so.b + head * so.h + t * so.t;
    TIn* y = h + bb * sy.b + head * sy.h + t * sy.t;

    // both rows are requested before the reductions, so their latencies overlap
    float v[NS][8], og[NS][8];
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int g = 2 * (64 * j + lane);   // first of this lane's two groups
        if (g + 1 < ng) {
            load8(x + 4 * g, v[j]);
            load8(o + 4 * g, og[j]);
        } else {
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                float (&vx)[4] = *reinterpret_cast<float(*)[4]>(&v[j][4 * hf]);
                float (&vo)[4] = *reinterpret_cast<float(*)[4]>(&og[j][4 * hf]);
                if (g + hf < ng) {
                    load4(x + 4 * (g + hf), vx);
                    load4(o + 4 * (g + hf), vo);
                } else {
                    vx[0] = vx[1] = vx[2] = vx[3] = 0.0f;
                    vo[0] = vo[1] = vo[2] = vo[3] = 0.0f;
                }
            }
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < NS; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) s += v[j][e];   // elements past the row are 0
    const float mean = rms ? 0.0f : wave_total(s) / static_cast<float>(DV);
    float ss = 0.0f;
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int g = 2 * (64 * j + lane);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float d = (g + e / 4 < ng) ? v[j][e] - mean : 0.0f;
            ss += d * d;
        }
    }
    const float inv = __builtin_amdgcn_rsqf(wave_total(ss) / static_cast<float>(DV) + eps);
    const float* w = weight ? weight + static_cast<int64_t>(head) * DV : nullptr;
    const float* b = bias ? bias + static_cast<int64_t>(head) * DV : nullptr;
#pragma unroll
    for (int j = 0; j < NS; ++j) {
        const int g = 2 * (64 * j + lane);
        if (g >= ng) continue;
        float out[8], wg[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f}, bg[8] = {};
        const bool full = g + 1 < ng;
        if (w) {
            if (full) load8(w + 4 * g, wg);
            else load4(w + 4 * g, *reinterpret_cast<float(*)[4]>(wg));
        }
        if (b) {
            if (full) load8(b + 4 * g, bg);
            else load4(b + 4 * g, *reinterpret_cast<float(*)[4]>(bg));
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float n = (v[j][e] - mean) * inv * wg[e] + bg[e];
            // sigmoid(o~) * n with the hardware exp and reciprocal (exp overflow gives 0)
            out[e] = n * __builtin_amdgcn_rcpf(1.0f + __expf(-og[j][e]));
        }
        if (full) store8(y + 4 * g, out);
        else store4(y + 4 * g, *reinterpret_cast<const float(*)[4]>(out));
    }
}

}  // namespace

hipError_t launch_output_norm(mlstm_dtype dt, const void* h_tilde, const void* o_pre, const float* weight,
                              const float* bias, float eps, int rms, int64_t rows, int NH, int T, int DV, void* h,
                              RowStrides so, RowStrides sy, hipStream_t stream) {
    constexpr int rpb = kNormThreads / 64;
    const dim3 grid(static_cast<unsigned>((rows + rpb - 1) / rpb));
    const int need = (DV + 511) / 512;
    auto go = [&](auto tag, auto ns) {
        using T_ = decltype(tag);
        hipLaunchKernelGGL((output_norm_kernel<T_, decltype(ns)::value>), grid, dim3(kNormThreads), 0, stream,
                           static_cast<const T_*>(h_tilde), static_cast<const T_*>(o_pre), weight, bias, eps, rms, rows,
                           NH, T, DV, static_cast<T_*>(h), so, sy);
    };
    auto by_width = [&](auto tag) {
        if (need <= 1) go(tag, std::integral_constant<int, 1>{});
        else if (need <= 2) go(tag, std::integral_constant<int, 2>{});
        else go(tag, std::integral_constant<int, kNormMaxSlabs>{});
    };
    if (dt == MLSTM_BF16) by_width(bf16_t{});
    else by_width(float{});
    return hipGetLastError();
}

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_output_norm)
#endif

}  // namespace mlstm
