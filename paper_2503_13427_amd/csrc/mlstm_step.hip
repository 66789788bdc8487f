// mlstm_step: one recurrent step of the mLSTM cell, fused into a single pass
// over the matrix memory (Sec. 2, Eqs. 2-5 with Eqs. 7-8; Sec. 3.1, "Fused
// Generation Kernels": the outer product, the dot products and the pointwise
// gate math run in one kernel so C is read once and written once).
//
// With enough sequences to fill the chip, one workgroup owns one (batch, head)
// sequence, so n and m may be updated in place: every element of C and n is read
// and written by the same thread, and m is written only after a barrier that
// follows every read of it.
//
// With few sequences (a decode step at batch 1 has 8), P workgroups split a
// sequence's DV columns so that the C stream runs on many CUs.  Each of them owns
// all DQK rows of its columns (the read-out C'^T q^ needs no exchange) and
// recomputes the scalar n'.q^ from n, which no workgroup of this launch writes;
// n' and m' are written by a second, small kernel that runs after it on the same
// stream, so an in-place update stays exact.
//
// The kernel is HBM-bound: C is streamed as float4 (128-bit) non-temporal loads
// and stores along DV; each thread walks a column group down the DQK rows with
// kBatch rows in flight, and the read-out C'^T q^ is reduced across the row
// groups in LDS.
//
// Output epilogue (mlstm_step_output).  When one workgroup owns a whole sequence and
// the read-out is reduced in LDS, the workgroup holds the full h~ row, so it can
// return the cell's hidden-state output instead (Eq. 6 with the output gate of
// Eq. 9): h = sigmoid(o~) * (Norm(h~) w + b), the headwise LayerNorm or RMSNorm
// taken over the row in fp32 from the unrounded h~ (two block reductions), and
// h~ never goes to memory.  Other launches write h~ and the output pass runs after.
#include "device_common.h"
#include "launch.h"

namespace mlstm {

constexpr int kStepThreads = 512;
constexpr int kBatch = 16;   // rows per pipeline stage

typedef float f4_t __attribute__((ext_vector_type(4)));

// Output epilogue of the fused launch (o == nullptr: the step returns h~)
template <typename TIn>
struct StepOut {
    const TIn* o;        // o~ [heads, DV]
    const float* w;      // [NH, DV] or nullptr (1)
    const float* b;      // [NH, DV] or nullptr (0)
    float eps;
    int rms;
    int NH;
};
constexpr int kOutPerThread = 4;   // h~ values a thread holds in the epilogue (DV <= 4 * 512)

__device__ __forceinline__ float block_sum(float x, float* wsum) {
    x = wave_sum(x);
    __syncthreads();   // wsum may still be read by the previous reduction
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = x;
    __syncthreads();
    float t = 0.0f;
#pragma unroll
    for (int w = 0; w < kStepThreads / 64; ++w) t += wsum[w];
    return t;
}

template <typename TIn>
__global__ void __launch_bounds__(kStepThreads)
step_kernel(const TIn* __restrict__ q, const TIn* __restrict__ k, const TIn* __restrict__ v,
            const float* __restrict__ ipre, const float* __restrict__ fpre,
            const float* C, const float* n, const float* m,
            int DQK, int DV, int P, TIn* __restrict__ h, float* C_out, float* n_out, float* m_out,
            StepOut<TIn> E) {
    extern __shared__ float smem[];
    float* qs = smem;                 // [DQK]   q / sqrt(DQK)
    float* iks = qs + DQK;            // [DQK]   i * k
    float* red = iks + DQK;           // [RG * DVs] partial read-outs
    __shared__ float wsum[kStepThreads / 64];

    // P workgroups per sequence, each owning DV / P columns (P = 1: the whole row and n, m)
    const int64_t head = blockIdx.x / P;
    const int part = blockIdx.x % P;
    const bool write_nm = (P == 1);
    const int DVs = DV / P;
    const int cv0 = part * DVs;       // first column of this workgroup
    const int tid = threadIdx.x;
    const int NC4 = DVs >> 2;         // float4 columns of this workgroup
    const int ROW4 = DV >> 2;         // float4 pitch of a C row
    const int RG = NC4 >= kStepThreads ? 1 : kStepThreads / NC4;
    const int rg = RG == 1 ? 0 : tid / NC4;    // row group: rows rg, rg + RG, ...
    const int c4_first = tid % NC4;            // first float4 column
    const int c4_stride = RG == 1 ? kStepThreads : NC4;
    const bool active = rg < RG;
    const int nrows = active ? (DQK - rg + RG - 1) / RG : 0;
    MLSTM_CHECK(cv0 + DVs <= DV && (DVs & 3) == 0 && (nrows == 0 || rg + (nrows - 1) * RG < DQK), kDbgStep);

    // C' = f C + (i k) v^T is streamed once (Eq. 3) with kBatch rows in flight per thread.
    // C_out may be C itself, so the compiler cannot hoist loads over stores; the next batch
    // is loaded explicitly before the current one is stored (disjoint rows, so the order is
    // exact).  The first batch is issued before the gate prologue, which it does not need.
    const f4_t* Ch = reinterpret_cast<const f4_t*>(C + head * static_cast<int64_t>(DQK) * DV + cv0);
    f4_t* Ch_out = reinterpret_cast<f4_t*>(C_out + head * static_cast<int64_t>(DQK) * DV + cv0);
    auto row = [&](int r) { return static_cast<int64_t>(rg + r * RG) * ROW4; };
    f4_t cur[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
        if (u < nrows) cur[u] = __builtin_nontemporal_load(&Ch[row(u) + c4_first]);
    // v of the first column group rides along with the first batch (it does not wait for the gates)
    const TIn* vh = v + head * DV + cv0;
    float vf[4] = {0.f, 0.f, 0.f, 0.f};
    if (active && c4_first < NC4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) vf[e] = io<TIn>::load(vh, 4 * c4_first + e);
    }

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
    float dot = 0.0f;
    for (int d = tid; d < DQK; d += kStepThreads) {
        const float qd = io<TIn>::load(qh, d) * qscale;
        const float ikd = ig * io<TIn>::load(kh, d);
        qs[d] = qd;
        iks[d] = ikd;
        const float nn = fg * nh[d] + ikd;
        if (write_nm) nh_out[d] = nn;
        dot += nn * qd;
    }
    dot = wave_sum(dot);
    if ((tid & 63) == 0) wsum[tid >> 6] = dot;
    __syncthreads();  // also orders every read of m[head] before the write below
    float qn = 0.0f;
#pragma unroll
    for (int w = 0; w < kStepThreads / 64; ++w) qn += wsum[w];
    const float inv = 1.0f / fmaxf(fabsf(qn), expf(-mnew));

    // s2 + s4: the C stream and num = C'^T q^ (Eqs. 3, 5)
    for (int c4 = c4_first; active && c4 < NC4; c4 += c4_stride) {
        if (c4 != c4_first) {
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                if (u < nrows) cur[u] = __builtin_nontemporal_load(&Ch[row(u) + c4]);
        }
        const bool first = (c4 == c4_first);
        const float v0 = first ? vf[0] : io<TIn>::load(vh, 4 * c4 + 0);
        const float v1 = first ? vf[1] : io<TIn>::load(vh, 4 * c4 + 1);
        const float v2 = first ? vf[2] : io<TIn>::load(vh, 4 * c4 + 2);
        const float v3 = first ? vf[3] : io<TIn>::load(vh, 4 * c4 + 3);
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
            TIn* hh = h + head * DV + cv0;
            io<TIn>::store(hh, 4 * c4 + 0, a0 * inv);
            io<TIn>::store(hh, 4 * c4 + 1, a1 * inv);
            io<TIn>::store(hh, 4 * c4 + 2, a2 * inv);
            io<TIn>::store(hh, 4 * c4 + 3, a3 * inv);
        } else {
            reinterpret_cast<float4*>(red)[rg * NC4 + c4] = make_float4(a0, a1, a2, a3);
        }
    }
    if (RG > 1 && !E.o) {
        __syncthreads();
        TIn* hh = h + head * DV + cv0;
        for (int j = tid; j < DVs; j += kStepThreads) {
            float s = 0.0f;
            for (int r = 0; r < RG; ++r) s += red[r * DVs + j];
            io<TIn>::store(hh, j, s * inv);
        }
    } else if (RG > 1) {
        // the output epilogue (launched only with P == 1, so DVs == DV <= kOutPerThread * 512)
        __syncthreads();
        float hv[kOutPerThread];
        float sum = 0.0f;
#pragma unroll
        for (int e = 0; e < kOutPerThread; ++e) {
            const int j = tid + e * kStepThreads;
            hv[e] = 0.0f;
            if (j < DV) {
                float s = 0.0f;
                for (int r = 0; r < RG; ++r) s += red[r * DV + j];
                hv[e] = s * inv;
                sum += hv[e];
            }
        }
        const float mean = E.rms ? 0.0f : block_sum(sum, wsum) / DV;
        float sq = 0.0f;
#pragma unroll
        for (int e = 0; e < kOutPerThread; ++e)
            if (tid + e * kStepThreads < DV) sq += (hv[e] - mean) * (hv[e] - mean);
        const float rstd = rsqrtf(block_sum(sq, wsum) / DV + E.eps);
        const int hd = static_cast<int>(head % E.NH);
        TIn* hh = h + head * DV;
        const TIn* oh = E.o + head * DV;
#pragma unroll
        for (int e = 0; e < kOutPerThread; ++e) {
            const int j = tid + e * kStepThreads;
            if (j < DV) {
                float y = (hv[e] - mean) * rstd;
                if (E.w) y *= E.w[static_cast<int64_t>(hd) * DV + j];
                if (E.b) y += E.b[static_cast<int64_t>(hd) * DV + j];
                const float gate = 1.0f / (1.0f + expf(-io<TIn>::load(oh, j)));
                io<TIn>::store(hh, j, gate * y);
            }
        }
    }
    if (write_nm && tid == 0) m_out[head] = mnew;
}

// n' = f n + i k and m' for each sequence (the split launch's second kernel); every element of
// n is read and written by one thread, and m' is written after the barrier that follows every
// read of m, so n_out and m_out may be n and m.
template <typename TIn>
__global__ void __launch_bounds__(256)
step_state_kernel(const TIn* __restrict__ k, const float* __restrict__ ipre, const float* __restrict__ fpre,
                  const float* n, const float* m, int DQK, float* n_out, float* m_out) {
    const int64_t head = blockIdx.x;
    const float mprev = m[head];
    const float a = logsigmoid(fpre[head]);
    const float it = ipre[head];
    const float mnew = fmaxf(a + mprev, it);
    const float fg = expf(a + mprev - mnew);
    const float ig = expf(it - mnew);
    for (int d = threadIdx.x; d < DQK; d += blockDim.x)
        n_out[head * DQK + d] = fg * n[head * DQK + d] + ig * io<TIn>::load(k + head * DQK, d);
    __syncthreads();
    if (threadIdx.x == 0) m_out[head] = mnew;
}

// Column splits per sequence: enough workgroups for the 256 CUs, at least 32 columns each (every
// row access then covers whole 128-byte lines).
static int step_splits(int heads, int DV) {
    int P = 1;
    while (static_cast<int64_t>(heads) * P < 256 && DV % (8 * P) == 0 && DV / (2 * P) >= 32) P *= 2;
    return P;
}

template <typename TIn>
static hipError_t launch_step_t(const void* q, const void* k, const void* v, const float* ipre, const float* fpre,
                                const float* C, const float* n, const float* m, int heads, int DQK, int DV, int P,
                                void* h, float* C_out, float* n_out, float* m_out, StepOut<TIn> E,
                                hipStream_t stream) {
    const size_t lds = step_lds_bytes(DQK, DV / P);
    const dim3 grid(static_cast<unsigned>(static_cast<int64_t>(heads) * P));
    hipLaunchKernelGGL(step_kernel<TIn>, grid, dim3(kStepThreads), lds, stream, static_cast<const TIn*>(q),
                       static_cast<const TIn*>(k), static_cast<const TIn*>(v), ipre, fpre, C, n, m, DQK, DV, P,
                       static_cast<TIn*>(h), C_out, n_out, m_out, E);
    if (P > 1)
        hipLaunchKernelGGL(step_state_kernel<TIn>, dim3(heads), dim3(256), 0, stream, static_cast<const TIn*>(k),
                           ipre, fpre, n, m, DQK, n_out, m_out);
    return hipGetLastError();
}

hipError_t launch_step(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                       const float* fpre, const float* C, const float* n, const float* m, int B, int NH,
                       int DQK, int DV, void* h, float* C_out, float* n_out, float* m_out,
                       hipStream_t stream) {
    const int heads = B * NH;
    const int P = step_splits(heads, DV);
    if (dt == MLSTM_BF16)
        return launch_step_t<bf16_t>(q, k, v, ipre, fpre, C, n, m, heads, DQK, DV, P, h, C_out, n_out, m_out,
                                     StepOut<bf16_t>{}, stream);
    return launch_step_t<float>(q, k, v, ipre, fpre, C, n, m, heads, DQK, DV, P, h, C_out, n_out, m_out,
                                StepOut<float>{}, stream);
}

bool step_output_fused(int B, int NH, int DQK, int DV) {
    (void)DQK;
    const int P = step_splits(B * NH, DV);
    const int NC4 = DV / 4;
    return P == 1 && NC4 < kStepThreads && DV <= kOutPerThread * kStepThreads;
}

hipError_t launch_step_output(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                              const float* fpre, const float* C, const float* n, const float* m, const void* o_pre,
                              const float* weight, const float* bias, float eps, int rms, int B, int NH, int DQK,
                              int DV, void* h, float* C_out, float* n_out, float* m_out, hipStream_t stream) {
    const int heads = B * NH;
    if (!step_output_fused(B, NH, DQK, DV)) {
        // the sequence's row is split over workgroups: h~ into h, then the output pass in place
        hipError_t e = launch_step(dt, q, k, v, ipre, fpre, C, n, m, B, NH, DQK, DV, h, C_out, n_out, m_out, stream);
        if (e != hipSuccess) return e;
        const RowStrides hm{static_cast<int64_t>(NH) * DV, DV, DV};
        return launch_output_norm(dt, h, o_pre, weight, bias, eps, rms, heads, NH, 1, DV, h, hm, hm, stream);
    }
    if (dt == MLSTM_BF16)
        return launch_step_t<bf16_t>(q, k, v, ipre, fpre, C, n, m, heads, DQK, DV, 1, h, C_out, n_out, m_out,
                                     StepOut<bf16_t>{static_cast<const bf16_t*>(o_pre), weight, bias, eps, rms, NH},
                                     stream);
    return launch_step_t<float>(q, k, v, ipre, fpre, C, n, m, heads, DQK, DV, 1, h, C_out, n_out, m_out,
                                StepOut<float>{static_cast<const float*>(o_pre), weight, bias, eps, rms, NH}, stream);
}

// LDS of one workgroup owning DVs columns: q^ and i k, then the partial read-outs of its row groups
size_t step_lds_bytes(int DQK, int DVs) {
    const int NC4 = DVs / 4;
    const int RG = NC4 >= kStepThreads ? 1 : kStepThreads / NC4;
    return sizeof(float) * (2 * static_cast<size_t>(DQK) + (RG > 1 ? static_cast<size_t>(RG) * DVs : 0));
}

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_step)
#endif

}  // namespace mlstm
