// Backward pass of the mLSTM cell (training mode) over the parallel form (Eq. 10), fp32 VALU.
//
// From the zero initial state, with b the prefix sums of logsig(f~), x_s = i~_s - b_s, the max
// state m_t = b_t + M_t (M_t = max(0, max_{s<=t} x_s), Eq. 2 from m_0 = 0) and q^ = q / sqrt(DQK),
// the forward output is h_t = N~_t / den_t with
//   F~_ts = exp(x_s - M_t)  (s <= t, every weight <= 1),   A~_ts = F~_ts (q^_t . k_s),
//   N~_t = sum_s A~_ts v_s,   D~_t = sum_s A~_ts,   den_t = max(|D~_t|, exp(-m_t)).
// Given dh, the chain rule gives (the derivation is the closed form the oracle pins):
//   dN~_t = dh_t / den_t,   dD~_t = -(dh_t . h_t) / den_t sign(D~_t) if |D~_t| > exp(-m_t), else 0,
//   W_ts = (dN~_t . v_s + dD~_t) F~_ts,
//   dq_t = sum_s W_ts k_s / sqrt(DQK),   dk_s = sum_t W_ts q^_t,   dv_s = sum_t A~_ts dN~_t,
//   di~_s = sum_t W_ts (q^_t . k_s),   P_t = dN~_t . N~_t + dD~_t D~_t,
//   df~_j = sigmoid(-f~_j) sum_{t >= j} (P_t - di~_t).
//
// Four launches per call:
//   gate pass    one thread per sequence: b, x, M, m into the workspace (a serial scan);
//   row pass     one workgroup per 16 rows t: a sweep over s <= t rebuilds N~ and D~ (so h),
//                gives dN~, dD~ and P (dN~ into the workspace); a second sweep accumulates dq;
//   column pass  one workgroup per 16 columns s: a sweep over t >= s accumulates dk, dv, di~;
//   forget pass  one thread per sequence: the reverse sum for df~.
// Tiles of 16 x 16 (t, s) pairs: one thread per pair for the dot products, then each thread of a
// row (or column) owns every 16th of its DV (or DQK) outputs.  LDS rows are padded by one float
// so that a row read across threads spreads over the banks.  Work is O(T^2 (DQK + DV)).
#include "device_common.h"
#include "launch.h"

namespace mlstm {
namespace {

constexpr int kBT = 16;                 // rows (or columns) per tile
constexpr int kBwdThreads = kBT * kBT;  // one thread per (t, s) pair of a tile
constexpr int kMaxDQK = 256;
constexpr int kMaxDV = 512;

struct BwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* ipre;
    const float* fpre;
    const float* dh;
    int T, DQK, DV;
    float* dq;
    float* dk;
    float* dv;
    float* dipre;
    float* dfpre;
    float* ws;          // per sequence: x, M, m, dD, P [T] then dN [T][DV]
};

__host__ __device__ inline int64_t ws_floats(int T, int DV) { return static_cast<int64_t>(T) * (5 + DV); }

// ---- gate pass ---------------------------------------------------------------------------------
__global__ void bwd_gate_kernel(BwdArgs A, int S) {
    const int s = blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S) return;
    const int T = A.T;
    float* w = A.ws + s * ws_floats(T, A.DV);
    float* x = w;
    float* M = w + T;
    float* m = w + 2 * T;
    const float* ib = A.ipre + static_cast<int64_t>(s) * T;
    const float* fb = A.fpre + static_cast<int64_t>(s) * T;
    float b = 0.0f, p = 0.0f;   // running prefix sum of logsig f~ and max(0, prefix max of x)
    for (int t = 0; t < T; ++t) {
        b += logsigmoid(fb[t]);
        const float xv = ib[t] - b;
        p = fmaxf(p, xv);
        x[t] = xv;
        M[t] = p;
        m[t] = b + p;
    }
}

// ---- row pass ----------------------------------------------------------------------------------
template <typename TIn>
__global__ void __launch_bounds__(kBwdThreads) bwd_row_kernel(BwdArgs A) {
    extern __shared__ float sm[];
    const int DQK = A.DQK, DV = A.DV, T = A.T;
    const int KP = DQK + 1, VP = DV + 1;   // LDS row pitches: rows read across threads hit distinct banks
    float* Qs = sm;                      // [kBT][KP] q^ rows of this tile
    float* Ks = Qs + kBT * KP;           // [kBT][KP] a tile of k
    float* Vs = Ks + kBT * KP;           // [kBT][VP] a tile of v
    float* dN = Vs + kBT * VP;           // [kBT][VP] dN~ of this tile's rows
    float* At = dN + kBT * VP;           // [kBT][kBT] A~ (sweep 1) or W (sweep 2)
    float* red = At + kBT * kBT;         // [kBT][kBT] row partial sums
    float* rowv = red + kBT * kBT;       // [kBT][4]   per row: M, m, dD, den
    const int ntile = (T + kBT - 1) / kBT;
    const int64_t seq = blockIdx.x / ntile;
    const int t0 = (blockIdx.x % ntile) * kBT;
    const int tid = threadIdx.x;
    // pair (row pr, column pc); for outputs, row pr and the columns j kBT + pc
    const int pr = tid / kBT, pc = tid % kBT;
    const TIn* q = static_cast<const TIn*>(A.q) + seq * T * DQK;
    const TIn* k = static_cast<const TIn*>(A.k) + seq * T * DQK;
    const TIn* v = static_cast<const TIn*>(A.v) + seq * T * DV;
    const float* wsq = A.ws + seq * ws_floats(T, DV);
    const float* xw = wsq;
    const float* Mw = wsq + T;
    const float* mw = wsq + 2 * T;
    float* dDw = const_cast<float*>(wsq) + 3 * T;
    float* Pw = const_cast<float*>(wsq) + 4 * T;
    float* dNw = const_cast<float*>(wsq) + 5 * T;
    const float qscale = rsqrtf(static_cast<float>(DQK));

    for (int e = tid; e < kBT * DQK; e += kBwdThreads) {
        const int r = e / DQK, d = e % DQK;
        Qs[r * KP + d] = (t0 + r < T) ? io<TIn>::load(q, static_cast<int64_t>(t0 + r) * DQK + d) * qscale : 0.0f;
    }
    if (tid < kBT) {
        const int t = t0 + tid;
        rowv[4 * tid + 0] = t < T ? Mw[t] : 0.0f;
        rowv[4 * tid + 1] = t < T ? mw[t] : 0.0f;
    }
    const int nv = DV / kBT;     // columns of v per thread (DV is a multiple of 16)
    const int nk = DQK / kBT;    // columns of k per thread
    float accN[kMaxDV / kBT];
#pragma unroll
    for (int j = 0; j < kMaxDV / kBT; ++j) accN[j] = 0.0f;
    float accD = 0.0f;
    const int last_tile = t0 / kBT;   // s tiles 0..last_tile hold s <= t for some row of this tile

    // sweep 1: N~ and D~ of the tile's rows
    for (int st = 0; st <= last_tile; ++st) {
        const int s0 = st * kBT;
        __syncthreads();   // the previous tile's Ks, Vs, At are no longer read
        for (int e = tid; e < kBT * DQK; e += kBwdThreads) {
            const int r = e / DQK, d = e % DQK;
            Ks[r * KP + d] = (s0 + r < T) ? io<TIn>::load(k, static_cast<int64_t>(s0 + r) * DQK + d) : 0.0f;
        }
        for (int e = tid; e < kBT * DV; e += kBwdThreads) {
            const int r = e / DV, d = e % DV;
            Vs[r * VP + d] = (s0 + r < T) ? io<TIn>::load(v, static_cast<int64_t>(s0 + r) * DV + d) : 0.0f;
        }
        __syncthreads();
        {
            const int t = t0 + pr, s = s0 + pc;
            float a = 0.0f;
            if (s <= t && t < T) {
                float dot = 0.0f;
                for (int d = 0; d < DQK; ++d) dot += Qs[pr * KP + d] * Ks[pc * KP + d];
                a = expf(xw[s] - rowv[4 * pr]) * dot;
            }
            At[pr * kBT + pc] = a;
        }
        __syncthreads();
        for (int s = 0; s < kBT; ++s) {
            const float a = At[pr * kBT + s];
            accD += (pc == 0) ? a : 0.0f;
#pragma unroll
            for (int j = 0; j < kMaxDV / kBT; ++j) if (j < nv) accN[j] += a * Vs[s * VP + j * kBT + pc];
        }
    }
    // dN~, dD~ and P per row: the row's 16 threads own nv columns each
    const int t = t0 + pr;
    const float* dhr = A.dh + (seq * T + (t < T ? t : 0)) * DV;
    if (pc == 0) red[pr * kBT] = accD;
    __syncthreads();
    const float Dt = red[pr * kBT];
    const float floor_t = expf(-rowv[4 * pr + 1]);
    const float den = fmaxf(fabsf(Dt), floor_t);
    float dhh = 0.0f, dnn = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxDV / kBT; ++j) if (j < nv) {
        const float g = t < T ? dhr[j * kBT + pc] : 0.0f;
        const float dn = g / den;
        dhh += g * (accN[j] / den);   // dh . h
        dnn += dn * accN[j];          // dN~ . N~
        dN[pr * VP + j * kBT + pc] = dn;
    }
    __syncthreads();
    red[pr * kBT + pc] = dhh;
    __syncthreads();
    if (pc == 0) {
        float sdh = 0.0f;
        for (int j = 0; j < kBT; ++j) sdh += red[pr * kBT + j];
        const float dD = (fabsf(Dt) > floor_t) ? -sdh / den * (Dt > 0.0f ? 1.0f : -1.0f) : 0.0f;
        rowv[4 * pr + 2] = dD;
    }
    __syncthreads();
    red[pr * kBT + pc] = dnn;
    __syncthreads();
    if (pc == 0 && t < T) {
        float sdn = 0.0f;
        for (int j = 0; j < kBT; ++j) sdn += red[pr * kBT + j];
        const float dD = rowv[4 * pr + 2];
        dDw[t] = dD;
        Pw[t] = sdn + dD * Dt;
    }
    if (t < T)
#pragma unroll
        for (int j = 0; j < kMaxDV / kBT; ++j) if (j < nv) dNw[static_cast<int64_t>(t) * DV + j * kBT + pc] = dN[pr * VP + j * kBT + pc];

    // sweep 2: dq_t = sum_s W_ts k_s / sqrt(DQK)
    float accQ[kMaxDQK / kBT];
#pragma unroll
    for (int j = 0; j < kMaxDQK / kBT; ++j) accQ[j] = 0.0f;
    for (int st = 0; st <= last_tile; ++st) {
        const int s0 = st * kBT;
        __syncthreads();
        for (int e = tid; e < kBT * DQK; e += kBwdThreads) {
            const int r = e / DQK, d = e % DQK;
            Ks[r * KP + d] = (s0 + r < T) ? io<TIn>::load(k, static_cast<int64_t>(s0 + r) * DQK + d) : 0.0f;
        }
        for (int e = tid; e < kBT * DV; e += kBwdThreads) {
            const int r = e / DV, d = e % DV;
            Vs[r * VP + d] = (s0 + r < T) ? io<TIn>::load(v, static_cast<int64_t>(s0 + r) * DV + d) : 0.0f;
        }
        __syncthreads();
        {
            const int s = s0 + pc;
            float w = 0.0f;
            if (s <= t && t < T) {
                float u = 0.0f;
                for (int d = 0; d < DV; ++d) u += dN[pr * VP + d] * Vs[pc * VP + d];
                w = (u + rowv[4 * pr + 2]) * expf(xw[s] - rowv[4 * pr]);
            }
            At[pr * kBT + pc] = w;
        }
        __syncthreads();
        for (int s = 0; s < kBT; ++s) {
            const float w = At[pr * kBT + s];
#pragma unroll
            for (int j = 0; j < kMaxDQK / kBT; ++j) if (j < nk) accQ[j] += w * Ks[s * KP + j * kBT + pc];
        }
    }
    if (t < T)
#pragma unroll
        for (int j = 0; j < kMaxDQK / kBT; ++j) if (j < nk) A.dq[(seq * T + t) * DQK + j * kBT + pc] = accQ[j] * qscale;
}

// ---- column pass -------------------------------------------------------------------------------
template <typename TIn>
__global__ void __launch_bounds__(kBwdThreads) bwd_col_kernel(BwdArgs A) {
    extern __shared__ float sm[];
    const int DQK = A.DQK, DV = A.DV, T = A.T;
    const int KP = DQK + 1, VP = DV + 1;   // LDS row pitches: rows read across threads hit distinct banks
    float* Ks = sm;                      // [kBT][KP] this tile's k
    float* Vs = Ks + kBT * KP;           // [kBT][VP] this tile's v
    float* Qs = Vs + kBT * VP;           // [kBT][KP] a tile of q^
    float* dN = Qs + kBT * KP;           // [kBT][VP] a tile of dN~
    float* Wt = dN + kBT * VP;           // [kBT][kBT] W, by (t, s)
    float* At = Wt + kBT * kBT;          // [kBT][kBT] A~, by (t, s)
    float* Gs = At + kBT * kBT;          // [kBT][kBT] W (q^ . k), by (t, s)
    float* rowv = Gs + kBT * kBT;        // [kBT][2]   per row t of the t tile: M, dD
    const int ntile = (T + kBT - 1) / kBT;
    const int64_t seq = blockIdx.x / ntile;
    const int s0 = (blockIdx.x % ntile) * kBT;
    const int tid = threadIdx.x;
    // pair (t row pr, s column pc); for outputs, column s0 + pr and the columns j kBT + pc
    const int pr = tid / kBT, pc = tid % kBT;
    const TIn* q = static_cast<const TIn*>(A.q) + seq * T * DQK;
    const TIn* k = static_cast<const TIn*>(A.k) + seq * T * DQK;
    const TIn* v = static_cast<const TIn*>(A.v) + seq * T * DV;
    const float* wsq = A.ws + seq * ws_floats(T, DV);
    const float* xw = wsq;
    const float* Mw = wsq + T;
    const float* dDw = wsq + 3 * T;
    const float* dNw = wsq + 5 * T;
    const float qscale = rsqrtf(static_cast<float>(DQK));

    for (int e = tid; e < kBT * DQK; e += kBwdThreads) {
        const int r = e / DQK, d = e % DQK;
        Ks[r * KP + d] = (s0 + r < T) ? io<TIn>::load(k, static_cast<int64_t>(s0 + r) * DQK + d) : 0.0f;
    }
    for (int e = tid; e < kBT * DV; e += kBwdThreads) {
        const int r = e / DV, d = e % DV;
        Vs[r * VP + d] = (s0 + r < T) ? io<TIn>::load(v, static_cast<int64_t>(s0 + r) * DV + d) : 0.0f;
    }
    const int nv = DV / kBT, nk = DQK / kBT;
    float accK[kMaxDQK / kBT], accV[kMaxDV / kBT];
#pragma unroll
    for (int j = 0; j < kMaxDQK / kBT; ++j) accK[j] = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxDV / kBT; ++j) accV[j] = 0.0f;
    float accI = 0.0f;
    const int s_own = s0 + pr;   // the column this thread accumulates for (outputs)
    for (int tt = s0 / kBT; tt < ntile; ++tt) {
        const int t0 = tt * kBT;
        __syncthreads();   // the previous tile's Qs, dN, Wt, At, Gs are no longer read
        for (int e = tid; e < kBT * DQK; e += kBwdThreads) {
            const int r = e / DQK, d = e % DQK;
            Qs[r * KP + d] = (t0 + r < T) ? io<TIn>::load(q, static_cast<int64_t>(t0 + r) * DQK + d) * qscale : 0.0f;
        }
        for (int e = tid; e < kBT * DV; e += kBwdThreads) {
            const int r = e / DV, d = e % DV;
            dN[r * VP + d] = (t0 + r < T) ? dNw[static_cast<int64_t>(t0 + r) * DV + d] : 0.0f;
        }
        if (tid < kBT) {
            const int t = t0 + tid;
            rowv[2 * tid + 0] = t < T ? Mw[t] : 0.0f;
            rowv[2 * tid + 1] = t < T ? dDw[t] : 0.0f;
        }
        __syncthreads();
        {
            const int t = t0 + pr, s = s0 + pc;
            float w = 0.0f, a = 0.0f, gq = 0.0f;
            if (s <= t && t < T && s < T) {
                float sqk = 0.0f, u = 0.0f;
                for (int d = 0; d < DQK; ++d) sqk += Qs[pr * KP + d] * Ks[pc * KP + d];
                for (int d = 0; d < DV; ++d) u += dN[pr * VP + d] * Vs[pc * VP + d];
                const float F = expf(xw[s] - rowv[2 * pr]);
                w = (u + rowv[2 * pr + 1]) * F;
                a = F * sqk;
                gq = w * sqk;
            }
            Wt[pr * kBT + pc] = w;
            At[pr * kBT + pc] = a;
            Gs[pr * kBT + pc] = gq;
        }
        __syncthreads();
        for (int r = 0; r < kBT; ++r) {
            const float w = Wt[r * kBT + pr];
            const float a = At[r * kBT + pr];
#pragma unroll
            for (int j = 0; j < kMaxDQK / kBT; ++j) if (j < nk) accK[j] += w * Qs[r * KP + j * kBT + pc];
#pragma unroll
            for (int j = 0; j < kMaxDV / kBT; ++j) if (j < nv) accV[j] += a * dN[r * VP + j * kBT + pc];
            accI += (pc == 0) ? Gs[r * kBT + pr] : 0.0f;
        }
    }
    if (s_own < T) {
#pragma unroll
        for (int j = 0; j < kMaxDQK / kBT; ++j) if (j < nk) A.dk[(seq * T + s_own) * DQK + j * kBT + pc] = accK[j];
#pragma unroll
        for (int j = 0; j < kMaxDV / kBT; ++j) if (j < nv) A.dv[(seq * T + s_own) * DV + j * kBT + pc] = accV[j];
        if (pc == 0) A.dipre[seq * T + s_own] = accI;
    }
}

// ---- forget pass -------------------------------------------------------------------------------
__global__ void bwd_forget_kernel(BwdArgs A, int S) {
    const int s = blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= S) return;
    const int T = A.T;
    const float* Pw = A.ws + s * ws_floats(T, A.DV) + 4 * T;
    const float* di = A.dipre + static_cast<int64_t>(s) * T;
    const float* fb = A.fpre + static_cast<int64_t>(s) * T;
    float* df = A.dfpre + static_cast<int64_t>(s) * T;
    float acc = 0.0f;
    for (int j = T - 1; j >= 0; --j) {
        acc += Pw[j] - di[j];
        df[j] = acc / (1.0f + expf(fb[j]));   // sigmoid(-f~)
    }
}

size_t row_lds(int DQK, int DV) {
    return sizeof(float) * (2 * kBT * (DQK + 1) + 2 * kBT * (DV + 1) + 2 * kBT * kBT + 4 * kBT);
}
size_t col_lds(int DQK, int DV) {
    return sizeof(float) * (2 * kBT * (DQK + 1) + 2 * kBT * (DV + 1) + 3 * kBT * kBT + 2 * kBT);
}

template <typename TIn>
hipError_t launch_typed(const BwdArgs& a, int S, hipStream_t stream) {
    const size_t lr = row_lds(a.DQK, a.DV), lc = col_lds(a.DQK, a.DV);
    static bool attr = false;
    if (!attr) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(bwd_row_kernel<TIn>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(row_lds(kMaxDQK, kMaxDV)));
        if (e != hipSuccess) return e;
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(bwd_col_kernel<TIn>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(col_lds(kMaxDQK, kMaxDV)));
        if (e != hipSuccess) return e;
        attr = true;
    }
    const int ntile = (a.T + kBT - 1) / kBT;
    const dim3 tiles(static_cast<unsigned>(static_cast<int64_t>(S) * ntile));
    const dim3 seqs(static_cast<unsigned>((S + 63) / 64));
    hipLaunchKernelGGL(bwd_gate_kernel, seqs, dim3(64), 0, stream, a, S);
    hipLaunchKernelGGL(bwd_row_kernel<TIn>, tiles, dim3(kBwdThreads), lr, stream, a);
    hipLaunchKernelGGL(bwd_col_kernel<TIn>, tiles, dim3(kBwdThreads), lc, stream, a);
    hipLaunchKernelGGL(bwd_forget_kernel, seqs, dim3(64), 0, stream, a, S);
    return hipGetLastError();
}

}  // namespace

bool parallel_bwd_supported(int DQK, int DV) {
    return DQK > 0 && DV > 0 && DQK % kBT == 0 && DV % kBT == 0 && DQK <= kMaxDQK && DV <= kMaxDV;
}

size_t parallel_bwd_workspace_bytes(int B, int NH, int T, int DV) {
    return static_cast<size_t>(B) * NH * static_cast<size_t>(ws_floats(T, DV)) * sizeof(float);
}

hipError_t launch_parallel_bwd(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                               const float* fpre, const float* dh, int B, int NH, int T, int DQK, int DV, float* dq,
                               float* dk, float* dv, float* dipre, float* dfpre, void* workspace, hipStream_t stream) {
    BwdArgs a{q, k, v, ipre, fpre, dh, T, DQK, DV, dq, dk, dv, dipre, dfpre, static_cast<float*>(workspace)};
    const int S = B * NH;
    return dt == MLSTM_BF16 ? launch_typed<bf16_t>(a, S, stream) : launch_typed<float>(a, S, stream);
}

}  // namespace mlstm
