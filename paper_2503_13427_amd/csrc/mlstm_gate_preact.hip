// Gate pre-activations of an mLSTM layer: the step right before the cell.
//
// Per token x (d values, bf16) and head h, the layer computes two scalar gate
// pre-activations, i~ = x . w_i[h] + b_i[h] and f~ = x . w_f[h] + b_f[h] (Eq. 11),
// passes both through the soft-cap a tanh(z / a) of Eq. 13, and, at the first token
// of a new document in a packed sequence, sets f~ = -inf: a forget gate of exactly
// zero, the state reset of App. B.  The result is written head-major, [B, NH, T]
// fp32, the layout mlstm_chunkwise_fwd and mlstm_step read.
//
// The projection is a skinny product: M = B T tokens by K = d by N = 2 NH gate
// columns.  It runs on bf16 MFMA (16x16x32, fp32 accumulation) so that the kernel
// stays bound by reading x once from HBM:
//   - a workgroup of NW waves owns MT 16-token tiles; each wave takes 1 / NW of K,
//     and the partial sums meet in LDS (four waves and four tiles for many tokens;
//     sixteen waves and one tile for a decode step, whose K walk is then short);
//   - both operands are 16-byte row reads: x rows as they are stored, the weights as
//     W^T [2 NH, d] (one row of d weights per gate column), which the caller stores
//     in that layout; W^T is small and stays in L2;
//   - the epilogue adds the bias, applies the cap and the border mask, and scatters
//     the 4 x 16 results of each lane group to the head-major outputs.
#include "device_common.h"
#include "launch.h"

namespace mlstm {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kGpUnroll = 4;          // k steps whose loads are issued together
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ f32x4_t mfma16(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0), static_cast<int>(bytes),
                                             kRsrcWord3);
}
// 16 bytes; reads past the resource's range return zeros
__device__ __forceinline__ u32x4_t bload128(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
    return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

struct GateArgs {
    const uint16_t* x;      // [M, d] bf16, M = B T
    const uint16_t* wt;     // [2 NH, d] bf16
    const float* bias;      // [2, NH] or NULL
    const uint8_t* border;  // [M] or NULL
    float cap;              // 0: no cap
    int64_t M;
    int T, d, NH;
    float* ipre;            // [B, NH, T]
    float* fpre;
};

// MT 16-token tiles per workgroup, NCT 16-column tiles of the 2 NH gate columns, NW waves.
template <int MT, int NCT, int NW>
__global__ void __launch_bounds__(64 * NW) gate_preact_kernel(GateArgs A) {
    constexpr int kThreadsW = 64 * NW;
    __shared__ f32x4_t red[NW][MT * NCT][64];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int l16 = lane & 15, g16 = lane >> 4;
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * (16 * MT);
    const int64_t rows = A.M - r0 < 16 * MT ? A.M - r0 : 16 * MT;
    // per-workgroup resources: the tile's x rows (rows beyond M read as zero) and all of W^T
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(A.x + r0 * A.d, static_cast<uint32_t>(rows * A.d * 2));
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(A.wt, static_cast<uint32_t>(2 * A.NH) * A.d * 2);

    const int kq = A.d / NW;         // this wave's share of K (a multiple of 32)
    const int k0 = wave * kq;
    MLSTM_CHECK(k0 + kq <= A.d && kq % 32 == 0, kDbgGatePreact);
    const int steps = kq / 32;
    f32x4_t acc[MT][NCT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) acc[mt][ct] = f32x4_t{};

    // lane (row or column l16, k group g16) reads the 8 consecutive k of its group
    uint32_t xo[MT], wo[NCT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) xo[mt] = static_cast<uint32_t>((16 * mt + l16) * A.d + k0 + 8 * g16) * 2;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) wo[ct] = static_cast<uint32_t>((16 * ct + l16) * A.d + k0 + 8 * g16) * 2;

    for (int s0 = 0; s0 < steps; s0 += kGpUnroll) {
        u32x4_t a[kGpUnroll][MT], b[kGpUnroll][NCT];
#pragma unroll
        for (int u = 0; u < kGpUnroll; ++u) {
            const uint32_t ko = static_cast<uint32_t>(32 * (s0 + u)) * 2;
            const bool ok = s0 + u < steps;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) a[u][mt] = ok ? bload128(rx, xo[mt] + ko) : u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) b[u][ct] = ok ? bload128(rw, wo[ct] + ko) : u32x4_t{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kGpUnroll; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) acc[mt][ct] = mfma16(a[u][mt], b[u][ct], acc[mt][ct]);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) red[wave][mt * NCT + ct][lane] = acc[mt][ct];
    __syncthreads();

    // lane group (tile mt, column tile ct, lane ln): column 16 ct + ln % 16, rows 4 (ln / 16) + 0..3
    const int ncol = 2 * A.NH;
    for (int it = tid; it < MT * NCT * 64; it += kThreadsW) {
        const int mc = it >> 6, ln = it & 63;
        const int mt = mc / NCT, ct = mc % NCT;
        const int j = 16 * ct + (ln & 15);
        if (j >= ncol) continue;
        f32x4_t z = red[0][mc][ln];
#pragma unroll
        for (int w = 1; w < NW; ++w) z += red[w][mc][ln];
        const bool forget = j >= A.NH;
        const int hd = forget ? j - A.NH : j;
        const float bj = A.bias ? A.bias[j] : 0.0f;
        float* out = forget ? A.fpre : A.ipre;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int64_t r = r0 + 16 * mt + 4 * (ln >> 4) + jj;
            if (r >= A.M) break;
            float g = z[jj] + bj;
            if (A.cap > 0.0f) g = A.cap * tanhf(g / A.cap);
            if (forget && A.border && A.border[r]) g = -INFINITY;
            const int64_t b = r / A.T, t = r - b * A.T;
            out[(b * A.NH + hd) * A.T + t] = g;
        }
    }
}

template <int MT, int NW>
void launch_mt(const GateArgs& a, int nct, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>((a.M + 16 * MT - 1) / (16 * MT)));
    const dim3 block(64 * NW);
    switch (nct) {
        case 1: hipLaunchKernelGGL((gate_preact_kernel<MT, 1, NW>), grid, block, 0, stream, a); break;
        case 2: hipLaunchKernelGGL((gate_preact_kernel<MT, 2, NW>), grid, block, 0, stream, a); break;
        case 3: hipLaunchKernelGGL((gate_preact_kernel<MT, 3, NW>), grid, block, 0, stream, a); break;
        default: hipLaunchKernelGGL((gate_preact_kernel<MT, 4, NW>), grid, block, 0, stream, a); break;
    }
}

}  // namespace

hipError_t launch_gate_preact(const void* x, const void* w_t, const float* bias, float cap, const uint8_t* border,
                              int B, int T, int d, int NH, float* ipre, float* fpre, hipStream_t stream) {
    GateArgs a{};
    a.x = static_cast<const uint16_t*>(x);
    a.wt = static_cast<const uint16_t*>(w_t);
    a.bias = bias;
    a.border = border;
    a.cap = cap;
    a.M = static_cast<int64_t>(B) * T;
    a.T = T;
    a.d = d;
    a.NH = NH;
    a.ipre = ipre;
    a.fpre = fpre;
    const int nct = (2 * NH + 15) / 16;
    // four tiles per workgroup once there are enough tokens to fill the chip with them; a decode
    // step's few tokens get sixteen waves on one tile (K walks of d / 512 steps)
    if (a.M >= 4096) launch_mt<4, 4>(a, nct, stream);
    else if (a.M <= 16 && d % (32 * 16) == 0) launch_mt<1, 16>(a, nct, stream);
    else launch_mt<1, 4>(a, nct, stream);
    return hipGetLastError();
}

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_gate_preact)
#endif

}  // namespace mlstm
