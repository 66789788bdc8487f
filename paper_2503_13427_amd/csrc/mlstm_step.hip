// mlstm_step: one recurrent step of the mLSTM cell, fused into a single pass
// over the matrix memory (Sec. 2, Eqs. 2-5 with Eqs. 7-8; Sec. 3.1, "Fused
// Generation Kernels": the outer product, the dot products and the pointwise
// gate math run in one kernel so C is read once and written once).
//
// One workgroup owns one (batch, head) sequence, so n and m may be updated in
// place: every element of C and n is read and written by the same thread, and
// m is written only after a barrier that follows every read of it.
//
// The kernel is HBM-bound: C is streamed as float4 (128-bit) non-temporal loads
// and stores along DV; each thread walks a column group down the DQK rows with
// kBatch rows in flight, and the read-out C'^T q^ is reduced across the row
// groups in LDS.
#include "device_common.h"
#include "launch.h"

namespace mlstm {

constexpr int kStepThreads = 512;
constexpr int kBatch = 16;   // rows per pipeline stage

typedef float f4_t __attribute__((ext_vector_type(4)));

template <typename TIn>
__global__ void __launch_bounds__(kStepThreads)
step_kernel(const TIn* __restrict__ q, const TIn* __restrict__ k, const TIn* __restrict__ v,
            const float* __restrict__ ipre, const float* __restrict__ fpre,
            const float* C, const float* n, const float* m,
            int DQK, int DV, TIn* __restrict__ h, float* C_out, float* n_out, float* m_out) {
    extern __shared__ float smem[];
    float* qs = smem;                 // [DQK]   q / sqrt(DQK)
    float* iks = qs + DQK;            // [DQK]   i * k
    float* red = iks + DQK;           // [RG * DV] partial read-outs
    __shared__ float wsum[kStepThreads / 64];

    const int64_t head = blockIdx.x;
    const int tid = threadIdx.x;
    const int NC4 = DV >> 2;
    const int RG = NC4 >= kStepThreads ? 1 : kStepThreads / NC4;
    const int rg = RG == 1 ? 0 : tid / NC4;    // row group: rows rg, rg + RG, ...
    const int c4_first = tid % NC4;            // first float4 column
    const int c4_stride = RG == 1 ? kStepThreads : NC4;
    const bool active = rg < RG;
    const int nrows = active ? (DQK - rg + RG - 1) / RG : 0;

    // C' = f C + (i k) v^T is streamed once (Eq. 3) with kBatch rows in flight per thread.
    // C_out may be C itself, so the compiler cannot hoist loads over stores; the next batch
    // is loaded explicitly before the current one is stored (disjoint rows, so the order is
    // exact).  The first batch is issued before the gate prologue, which it does not need.
    const f4_t* Ch = reinterpret_cast<const f4_t*>(C + head * static_cast<int64_t>(DQK) * DV);
    f4_t* Ch_out = reinterpret_cast<f4_t*>(C_out + head * static_cast<int64_t>(DQK) * DV);
    auto row = [&](int r) { return static_cast<int64_t>(rg + r * RG) * NC4; };
    f4_t cur[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
        if (u < nrows) cur[u] = __builtin_nontemporal_load(&Ch[row(u) + c4_first]);

    // s1: scalar gates (Eqs. 2, 7, 8), computed redundantly by every thread
    const float mprev = m[head];
    const float a = logsigmoid(fpre[head]);
    const float it = ipre[head];
    const float mnew = fmaxf(a + mprev, it);
    const float fg = expf(a + mprev - mnew);
    const float ig = expf(it - mnew);
    const float qscale = rsqrtf(static_cast<float>(DQK));

    const TIn* qh = q + head * DQK;
    const TIn* kh = k + head * DQK;
    const float* nh = n + head * DQK;
    float* nh_out = n_out + head * DQK;

    // s3: n' = f n + i k, and the partial n'.q^ (Eq. 4, denominator of Eq. 5)
    float part = 0.0f;
    for (int d = tid; d < DQK; d += kStepThreads) {
        const float qd = io<TIn>::load(qh, d) * qscale;
        const float ikd = ig * io<TIn>::load(kh, d);
        qs[d] = qd;
        iks[d] = ikd;
        const float nn = fg * nh[d] + ikd;
        nh_out[d] = nn;
        part += nn * qd;
    }
    part = wave_sum(part);
    if ((tid & 63) == 0) wsum[tid >> 6] = part;
    __syncthreads();  // also orders every read of m[head] before the write below
    float qn = 0.0f;
#pragma unroll
    for (int w = 0; w < kStepThreads / 64; ++w) qn += wsum[w];
    const float inv = 1.0f / fmaxf(fabsf(qn), expf(-mnew));

    // s2 + s4: the C stream and num = C'^T q^ (Eqs. 3, 5)
    const TIn* vh = v + head * DV;
    for (int c4 = c4_first; active && c4 < NC4; c4 += c4_stride) {
        if (c4 != c4_first) {
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                if (u < nrows) cur[u] = __builtin_nontemporal_load(&Ch[row(u) + c4]);
        }
        const float v0 = io<TIn>::load(vh, 4 * c4 + 0), v1 = io<TIn>::load(vh, 4 * c4 + 1);
        const float v2 = io<TIn>::load(vh, 4 * c4 + 2), v3 = io<TIn>::load(vh, 4 * c4 + 3);
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
        for (int r0 = 0; r0 < nrows; r0 += kBatch) {
            f4_t nxt[kBatch];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int r = r0 + kBatch + u;
                if (r < nrows) nxt[u] = __builtin_nontemporal_load(&Ch[row(r) + c4]);
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int r = r0 + u;
                if (r < nrows) {
                    const int d = rg + r * RG;
                    f4_t c = cur[u];
                    const float ikd = iks[d];
                    c.x = fg * c.x + ikd * v0;
                    c.y = fg * c.y + ikd * v1;
                    c.z = fg * c.z + ikd * v2;
                    c.w = fg * c.w + ikd * v3;
                    __builtin_nontemporal_store(c, &Ch_out[row(r) + c4]);
                    const float qd = qs[d];
                    a0 += qd * c.x;
                    a1 += qd * c.y;
                    a2 += qd * c.z;
                    a3 += qd * c.w;
                }
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u) cur[u] = nxt[u];
        }
        if (RG == 1) {
            // s5: h = num / max(|n'.q^|, exp(-m'))
            TIn* hh = h + head * DV;
            io<TIn>::store(hh, 4 * c4 + 0, a0 * inv);
            io<TIn>::store(hh, 4 * c4 + 1, a1 * inv);
            io<TIn>::store(hh, 4 * c4 + 2, a2 * inv);
            io<TIn>::store(hh, 4 * c4 + 3, a3 * inv);
        } else {
            reinterpret_cast<float4*>(red)[rg * NC4 + c4] = make_float4(a0, a1, a2, a3);
        }
    }
    if (RG > 1) {
        __syncthreads();
        TIn* hh = h + head * DV;
        for (int j = tid; j < DV; j += kStepThreads) {
            float s = 0.0f;
            for (int r = 0; r < RG; ++r) s += red[r * DV + j];
            io<TIn>::store(hh, j, s * inv);
        }
    }
    if (tid == 0) m_out[head] = mnew;
}

hipError_t launch_step(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                       const float* fpre, const float* C, const float* n, const float* m, int B, int NH,
                       int DQK, int DV, void* h, float* C_out, float* n_out, float* m_out,
                       hipStream_t stream) {
    const int heads = B * NH;
    const int NC4 = DV / 4;
    const int RG = NC4 >= kStepThreads ? 1 : kStepThreads / NC4;
    const size_t lds = sizeof(float) * (2 * static_cast<size_t>(DQK) + (RG > 1 ? static_cast<size_t>(RG) * DV : 0));
    if (dt == MLSTM_BF16) {
        hipLaunchKernelGGL(step_kernel<bf16_t>, dim3(heads), dim3(kStepThreads), lds, stream,
                           static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                           static_cast<const bf16_t*>(v), ipre, fpre, C, n, m, DQK, DV,
                           static_cast<bf16_t*>(h), C_out, n_out, m_out);
    } else {
        hipLaunchKernelGGL(step_kernel<float>, dim3(heads), dim3(kStepThreads), lds, stream,
                           static_cast<const float*>(q), static_cast<const float*>(k),
                           static_cast<const float*>(v), ipre, fpre, C, n, m, DQK, DV,
                           static_cast<float*>(h), C_out, n_out, m_out);
    }
    return hipGetLastError();
}

size_t step_lds_bytes(int DQK, int DV) {
    const int NC4 = DV / 4;
    const int RG = NC4 >= kStepThreads ? 1 : kStepThreads / NC4;
    return sizeof(float) * (2 * static_cast<size_t>(DQK) + (RG > 1 ? static_cast<size_t>(RG) * DV : 0));
}

}  // namespace mlstm
