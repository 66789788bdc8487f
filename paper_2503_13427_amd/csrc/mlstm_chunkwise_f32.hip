// Chunkwise-parallel mLSTM forward, fp32 VALU kernel for small heads.
//
// The chunkwise form (Sec. 2, "Training Mode") processes the sequence in
// chunks of L tokens: within a chunk the outputs come from a causal,
// gate-weighted L x L matrix (the intra-chunk part), and the chunk's entry
// state carries everything before it (the inter-chunk part).  The sub-steps
// follow App. D.1: chunkwise gates (prefix sums of logsig f~), gates and max
// state, inter-chunk numerator and denominator, gate matrix, gated logits,
// intra-chunk numerator and denominator, output combination.
//
// Stabiliser bookkeeping.  With b_tau the in-chunk prefix sum of logsig f~
// and p_tau = max_{sig <= tau}(i~_sig - b_sig), the max state of Eq. 2 is
// m_tau = b_tau + M_tau with M_tau = max(m_prev, p_tau).  Every exponent is
// then written as a difference against M, so it is <= 0 by construction:
//   gate matrix      D[tau,sig] = exp((i~_sig - b_sig) - M_tau)     (sig <= tau)
//   entry-state term             exp(m_prev - M_tau)
//   state decay                  exp(m_prev - M_L)
//   key weights      w_tau     = exp((i~_tau - b_tau) - M_L)
//   floor                        exp(-(b_tau + M_tau))
// and the chunk's exit max state is b_L + M_L.
//
// A forget gate of exactly zero (f~ = -inf, a document border) restarts the state.  The prefix
// sum b skips the restart token, each row keeps its last restart R_tau, the gate matrix keeps
// only R_tau <= sig <= tau, p restarts at R_tau, a row at or after a restart has no entry-state
// term, and a chunk that holds a restart drops its entry state (decay 0) and weights only the
// keys from its last restart on.
//
// One workgroup owns a (sequence, dv tile) pair and walks the chunks in order
// with its C tile, n and m in LDS.  Storage and the gate arithmetic are fp32; q, k, v may be
// fp32 or bf16.  The dot products (logits, read-outs, state updates) accumulate in fp64, so a
// row whose sum cancels keeps the accuracy of its fp32 operands rather than of an fp32 sum.  This kernel is the fp32 path and the reference schedule; the bf16
// xLSTM-7B head shape runs on the MFMA kernel.
#include "device_common.h"
#include "launch.h"

namespace mlstm {

constexpr int kF32Threads = 256;
constexpr size_t kF32LdsBudget = 64 * 1024;

static size_t f32_lds_floats(int DQK, int DVT, int L) {
    return static_cast<size_t>(DQK) * DVT + DQK + 2 * static_cast<size_t>(L) * DQK +
           static_cast<size_t>(L) * DVT + static_cast<size_t>(L) * L + 8 * static_cast<size_t>(L) + 8;
}

int chunk_f32_tile(int DQK, int DV, int L) {
    for (int dvt = DV; dvt >= 1; dvt >>= 1) {
        if (DV % dvt) continue;
        if (f32_lds_floats(DQK, dvt, L) * sizeof(float) <= kF32LdsBudget) return dvt;
        if (dvt & 1) break;
    }
    return 0;
}

template <typename TIn>
__global__ void __launch_bounds__(kF32Threads)
chunk_f32_kernel(const TIn* __restrict__ q, const TIn* __restrict__ k, const TIn* __restrict__ v,
                 const float* __restrict__ ipre, const float* __restrict__ fpre,
                 const float* __restrict__ C0, const float* __restrict__ n0, const float* __restrict__ m0,
                 int T, int DQK, int DV, int L, int DVT, TIn* __restrict__ h, float* __restrict__ CT,
                 float* __restrict__ nT, float* __restrict__ mT) {
    extern __shared__ float smem[];
    float* Cs = smem;                                   // [DQK][DVT]
    float* ns = Cs + DQK * DVT;                         // [DQK]
    float* Qs = ns + DQK;                               // [L][DQK]   q / sqrt(DQK)
    float* Ks = Qs + L * DQK;                           // [L][DQK]
    float* Vs = Ks + L * DQK;                           // [L][DVT]
    float* Sm = Vs + L * DVT;                           // [L][L]     gated logits S~
    float* g_ib = Sm + L * L;                           // [L]  i~ - b
    float* g_M = g_ib + L;                              // [L]  M_tau
    float* g_inter = g_M + L;                           // [L]  exp(m_prev - M_tau)
    float* g_floor = g_inter + L;                       // [L]  exp(-(b_tau + M_tau))
    float* g_w = g_floor + L;                           // [L]  key weights
    float* g_den = g_w + L;                             // [L]  1 / max(|den|, floor)
    float* g_sc = g_den + 2 * L;                        // scalars: [0] m_prev, [1] decay
    float* g_R = g_sc + 8;                              // [L]  last restart at or before the row (-1: none)

    const int ntiles = DV / DVT;
    const int64_t seq = blockIdx.x / ntiles;
    const int tile = blockIdx.x % ntiles;
    MLSTM_CHECK(ntiles * DVT == DV && L <= T + L, kDbgChunkF32);
    const int v0 = tile * DVT;
    const int tid = threadIdx.x;
    const float qscale = rsqrtf(static_cast<float>(DQK));

    // initial state (zero state has m0 = 0)
    for (int e = tid; e < DQK * DVT; e += kF32Threads) {
        const int d = e / DVT, j = e % DVT;
        Cs[e] = C0 ? C0[(seq * DQK + d) * DV + v0 + j] : 0.0f;
    }
    for (int d = tid; d < DQK; d += kF32Threads) ns[d] = n0 ? n0[seq * DQK + d] : 0.0f;
    if (tid == 0) g_sc[0] = m0 ? m0[seq] : 0.0f;
    __syncthreads();

    const TIn* qb = q + seq * static_cast<int64_t>(T) * DQK;
    const TIn* kb = k + seq * static_cast<int64_t>(T) * DQK;
    const TIn* vb = v + seq * static_cast<int64_t>(T) * DV;
    TIn* hb = h + seq * static_cast<int64_t>(T) * DV;

    for (int t0 = 0; t0 < T; t0 += L) {
        // rows lc..L-1 of a partial last chunk are neutral tokens: zero q, k, v, no input
        // (x = -inf) and no decay, so they leave the state unchanged; their h is not written
        const int lc = min(L, T - t0);
        // stage the chunk
        for (int e = tid; e < L * DQK; e += kF32Threads) {
            const bool ok = e < lc * DQK;
            Qs[e] = ok ? io<TIn>::load(qb, static_cast<int64_t>(t0) * DQK + e) * qscale : 0.0f;
            Ks[e] = ok ? io<TIn>::load(kb, static_cast<int64_t>(t0) * DQK + e) : 0.0f;
        }
        for (int e = tid; e < L * DVT; e += kF32Threads) {
            const int t = e / DVT, j = e % DVT;
            Vs[e] = t < lc ? io<TIn>::load(vb, static_cast<int64_t>(t0 + t) * DV + v0 + j) : 0.0f;
        }
        // chunkwise gates and max state: a short serial scan (L <= 64)
        if (tid == 0) {
            const float mprev = g_sc[0];
            const float* ib = ipre + seq * static_cast<int64_t>(T) + t0;
            const float* fb = fpre + seq * static_cast<int64_t>(T) + t0;
            float b = 0.0f, p = -INFINITY;
            int R = -1;
            for (int t = 0; t < L; ++t) {
                const float lg = t < lc ? logsigmoid(fb[t]) : 0.0f;
                if (lg == -INFINITY) {
                    R = t;
                    p = -INFINITY;
                } else {
                    b += lg;
                }
                const float x = t < lc ? ib[t] - b : -INFINITY;
                p = fmaxf(p, x);
                const float M = R >= 0 ? p : fmaxf(mprev, p);
                g_ib[t] = x;
                g_M[t] = M;
                g_R[t] = static_cast<float>(R);
                g_inter[t] = (R >= 0 || M == -INFINITY) ? 0.0f : expf(mprev - M);
                g_floor[t] = expf(-(b + M));
            }
            const float ML = g_M[L - 1];
            for (int t = 0; t < L; ++t) g_w[t] = (t < R || ML == -INFINITY) ? 0.0f : expf(g_ib[t] - ML);
            g_sc[1] = (R >= 0 || ML == -INFINITY) ? 0.0f : expf(mprev - ML);
            g_sc[0] = b + ML;  // exit max state m_k
        }
        __syncthreads();

        // gated logits S~ = (Q^ K^T) * D, causal
        for (int e = tid; e < L * L; e += kF32Threads) {
            const int t = e / L, s = e % L;
            float val = 0.0f;
            if (s <= t && s >= static_cast<int>(g_R[t]) && g_M[t] != -INFINITY) {
                double acc = 0.0;
                for (int d = 0; d < DQK; ++d) acc += static_cast<double>(Qs[t * DQK + d]) * Ks[s * DQK + d];
                val = static_cast<float>(acc) * expf(g_ib[s] - g_M[t]);
            }
            Sm[e] = val;
        }
        __syncthreads();

        // denominators: exp(m_prev - M) q^.n + rowsum(S~), floored
        for (int t = tid; t < L; t += kF32Threads) {
            double qn = 0.0;
            for (int d = 0; d < DQK; ++d) qn += static_cast<double>(Qs[t * DQK + d]) * ns[d];
            double rs = 0.0;
            for (int s = 0; s <= t; ++s) rs += Sm[t * L + s];
            const float den = static_cast<float>(g_inter[t] * qn + rs);
            g_den[t] = 1.0f / fmaxf(fabsf(den), g_floor[t]);
        }
        __syncthreads();

        // numerators and output combination
        for (int e = tid; e < lc * DVT; e += kF32Threads) {
            const int t = e / DVT, j = e % DVT;
            double inter = 0.0;
            for (int d = 0; d < DQK; ++d) inter += static_cast<double>(Qs[t * DQK + d]) * Cs[d * DVT + j];
            double intra = 0.0;
            for (int s = 0; s <= t; ++s) intra += static_cast<double>(Sm[t * L + s]) * Vs[s * DVT + j];
            io<TIn>::store(hb, static_cast<int64_t>(t0 + t) * DV + v0 + j,
                           static_cast<float>((g_inter[t] * inter + intra) * g_den[t]));
        }
        __syncthreads();

        // state update: C = decay C + (w K)^T V, n = decay n + K^T w
        const float decay = g_sc[1];
        for (int e = tid; e < DQK * DVT; e += kF32Threads) {
            const int d = e / DVT, j = e % DVT;
            double acc = 0.0;
            for (int t = 0; t < L; ++t) acc += static_cast<double>(g_w[t] * Ks[t * DQK + d]) * Vs[t * DVT + j];
            Cs[e] = static_cast<float>(decay * static_cast<double>(Cs[e]) + acc);
        }
        for (int d = tid; d < DQK; d += kF32Threads) {
            double acc = 0.0;
            for (int t = 0; t < L; ++t) acc += static_cast<double>(g_w[t]) * Ks[t * DQK + d];
            ns[d] = static_cast<float>(decay * static_cast<double>(ns[d]) + acc);
        }
        __syncthreads();
    }

    // final state
    for (int e = tid; e < DQK * DVT; e += kF32Threads) {
        const int d = e / DVT, j = e % DVT;
        CT[(seq * DQK + d) * DV + v0 + j] = Cs[e];
    }
    if (tile == 0) {
        for (int d = tid; d < DQK; d += kF32Threads) nT[seq * DQK + d] = ns[d];
        if (tid == 0) mT[seq] = g_sc[0];
    }
}

hipError_t launch_chunk_f32(mlstm_dtype dt, const ChunkArgs& a, hipStream_t stream) {
    const int dvt = chunk_f32_tile(a.DQK, a.DV, a.L);
    const size_t lds = f32_lds_floats(a.DQK, dvt, a.L) * sizeof(float);
    const dim3 grid(static_cast<unsigned>(a.B * a.NH * (a.DV / dvt)));
    if (dt == MLSTM_BF16) {
        hipLaunchKernelGGL(chunk_f32_kernel<bf16_t>, grid, dim3(kF32Threads), lds, stream,
                           static_cast<const bf16_t*>(a.q), static_cast<const bf16_t*>(a.k),
                           static_cast<const bf16_t*>(a.v), a.ipre, a.fpre, a.C0, a.n0, a.m0, a.T, a.DQK,
                           a.DV, a.L, dvt, static_cast<bf16_t*>(a.h), a.CT, a.nT, a.mT);
    } else {
        hipLaunchKernelGGL(chunk_f32_kernel<float>, grid, dim3(kF32Threads), lds, stream,
                           static_cast<const float*>(a.q), static_cast<const float*>(a.k),
                           static_cast<const float*>(a.v), a.ipre, a.fpre, a.C0, a.n0, a.m0, a.T, a.DQK,
                           a.DV, a.L, dvt, static_cast<float*>(a.h), a.CT, a.nT, a.mT);
    }
    return hipGetLastError();
}

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_chunk_f32)
#endif

}  // namespace mlstm
