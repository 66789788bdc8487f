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
//   gate pass    one wave per sequence: b, x, M, m into the workspace (wave scans);
//   row pass     one workgroup per 16 rows t: a sweep over s <= t rebuilds N~ and D~ (so h),
//                gives dN~, dD~ and P (dN~ into the workspace); a second sweep accumulates dq;
//   column pass  one workgroup per 16 columns s: a sweep over t >= s accumulates dk, dv, di~;
//   forget pass  one wave per sequence: the reverse sum for df~.
// Tiles of 16 x 16 (t, s) pairs: one thread per pair for the dot products, then each thread of a
// row (or column) owns every 16th of its DV (or DQK) outputs.  LDS rows are padded by one float
// so that a row read across threads spreads over the banks.  Work is O(T^2 (DQK + DV)).
#include <utility>

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
    float* ws;          // per sequence: x, M, m, dD, P [T], then from dn_off(T) dN [T][DV]
};

// dN starts on a 16-byte boundary (the passes stage it with 16-byte loads); DV is a multiple of 16,
// so every sequence's block is a multiple of four floats too
__host__ __device__ inline int64_t dn_off(int T) { return (5 * static_cast<int64_t>(T) + 3) & ~int64_t(3); }
__host__ __device__ inline int64_t ws_floats(int T, int DV) { return dn_off(T) + static_cast<int64_t>(T) * DV; }

// ---- gate pass ---------------------------------------------------------------------------------
// Inclusive scans over a wave (shift-and-combine, 6 steps).
__device__ __forceinline__ float wave_scan_sum(float x, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    return x;
}
__device__ __forceinline__ float wave_scan_max(float x, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float y = __shfl_up(x, o, 64);
        if (lane >= o) x = fmaxf(x, y);
    }
    return x;
}
constexpr int kScanBatch = 8;   // 64-token steps of a scan whose loads are issued together

// one wave per sequence, 64 tokens per step: b, x = i~ - b, M = max(0, prefix max of x), m = b + M
__global__ void bwd_gate_kernel(BwdArgs A, int S) {
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    const int T = A.T;
    float* w = A.ws + s * ws_floats(T, A.DV);
    float* x = w;
    float* M = w + T;
    float* m = w + 2 * T;
    const float* ib = A.ipre + static_cast<int64_t>(s) * T;
    const float* fb = A.fpre + static_cast<int64_t>(s) * T;
    float b_carry = 0.0f, p_carry = 0.0f;
    for (int tb = 0; tb < T; tb += 64 * kScanBatch) {
        float fv[kScanBatch], iv[kScanBatch];
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u) {
            const int t = tb + 64 * u + lane;
            fv[u] = t < T ? fb[t] : 0.0f;
            iv[u] = t < T ? ib[t] : 0.0f;
        }
        // the sum scans of the batch do not depend on one another: run them first, then add the
        // carries in order (the same roundings as one scan after another)
        float ls[kScanBatch], lt[kScanBatch];
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u) {
            const int t = tb + 64 * u + lane;
            ls[u] = wave_scan_sum(t < T ? logsigmoid(fv[u]) : 0.0f, lane);
            lt[u] = __shfl(ls[u], 63, 64);
        }
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u) {
            const int t = tb + 64 * u + lane;
            const bool ok = t < T;
            const float b = b_carry + ls[u];
            const float xv = ok ? iv[u] - b : -INFINITY;
            const float p = fmaxf(p_carry, wave_scan_max(xv, lane));
            if (ok) {
                x[t] = xv;
                M[t] = p;
                m[t] = b + p;
            }
            b_carry += lt[u];
            p_carry = __shfl(p, 63, 64);
        }
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
    MLSTM_CHECK(t0 < T && DQK % 16 == 0 && DV % 16 == 0, kDbgParallelBwd);
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
    float* dNw = const_cast<float*>(wsq) + dn_off(T);
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
    const float* dNw = wsq + dn_off(T);
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

// ---- MFMA row and column passes (instantiated head shapes) ------------------------------------
//
// The same passes with the tile products on fp32 MFMA 16x16x4 (lane l: A[l % 16][l / 16],
// B[l / 16][l % 16], D[4 (l / 16) + j][l % 16]).  Per 16 x 16 tile of (t, s) pairs:
//   - the logits S = Q^ K^T (or U = dN~ V^T) are split over the four waves along the contraction
//     and their partial tiles summed through LDS; the operand that stays fixed over a sweep (the
//     row pass's q^ and dN~ rows, the column pass's k and v rows) is held in registers;
//   - the k, v and q tiles stay in the input type in LDS, so with bf16 inputs a row-pass
//     workgroup takes 34 KB of LDS and a column-pass workgroup 52 KB (dN~ stays fp32), and
//     three share a CU;
//   - one thread per pair applies the gates (F~, the causal mask) and writes the operand tile;
//   - the accumulating products (N~ += A~ V, dq += W K; dk += W^T Q^, dv += A~^T dN~) give each
//     wave a quarter of the output columns, one 16 x 16 accumulator per 16 columns.
// fp32 LDS rows are padded to a pitch of 4 (mod 32) floats.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
constexpr int kMaxNT = kMaxDV / 64;     // 16-column output tiles per wave, at most (DV = 512)
constexpr int kTP = kBT + 4;            // pitch of a 16 x 16 operand tile

__device__ __forceinline__ f32x4_t mfma4(float a, float b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <typename TIn> struct Vec16;
template <> struct Vec16<float> {
    static constexpr int N = 4;
    typedef float4 type;
    static __device__ __forceinline__ void widen(const type& v, float (&o)[4]) { o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w; }
};
template <> struct Vec16<bf16_t> {
    static constexpr int N = 8;
    typedef uint4 type;
    static __device__ __forceinline__ void widen(const type& v, float (&o)[8]) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[2 * i] = __uint_as_float(w[i] << 16);
            o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
};
template <typename TIn, int NMAX = kMaxDV>
__device__ __forceinline__ void stage_rows(float* dst, int pitch, const TIn* src, int r0, int nrows_total, int n,
                                           float scale, int tid) {
    typedef Vec16<TIn> V;
    constexpr int kMaxPer = (kBT * NMAX / V::N + kBwdThreads - 1) / kBwdThreads;   // vectors per thread, at most
    const int nvec = kBT * n / V::N;
    typename V::type buf[kMaxPer];
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        const int idx = tid + kBwdThreads * i;
        const int r = (idx * V::N) / n;
        if (idx < nvec && r0 + r < nrows_total)
            buf[i] = reinterpret_cast<const typename V::type*>(src + static_cast<int64_t>(r0) * n)[idx];
    }
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        const int idx = tid + kBwdThreads * i;
        if (idx < nvec) {
            const int e = idx * V::N, r = e / n, d = e % n;
            float o[V::N];
            if (r0 + r < nrows_total) {
                V::widen(buf[i], o);
            } else {
#pragma unroll
                for (int j = 0; j < V::N; ++j) o[j] = 0.0f;
            }
#pragma unroll
            for (int j = 0; j < V::N; ++j) dst[r * pitch + d + j] = o[j] * scale;
        }
    }
}
// the same for fp32 rows of the workspace
template <int NMAX>
__device__ __forceinline__ void stage_rows_f32(float* dst, int pitch, const float* src, int r0, int nrows_total, int n,
                                               int tid) {
    stage_rows<float, NMAX>(dst, pitch, src, r0, nrows_total, n, 1.0f, tid);
}

// k, v and q tiles stay in the input type in LDS (half the bytes for bf16, so more workgroups
// share a CU); rows beyond T are zero.  A bf16 row pitch of n + 8 elements keeps the 16-byte
// stores aligned and the row and column reads of the passes at most 2-way bank-conflicted.
template <typename TIn> constexpr int lds_pad() { return sizeof(TIn) == 2 ? 8 : 4; }
__device__ __forceinline__ float lds_ld(const float* p, int i) { return p[i]; }
__device__ __forceinline__ float lds_ld(const bf16_t* p, int i) { return bf16_to_f32(p[i].bits); }
template <typename TIn, int NMAX>
__device__ __forceinline__ void stage_raw(TIn* dst, int pitch, const TIn* src, int r0, int nrows_total, int n,
                                          int tid) {
    typedef typename Vec16<TIn>::type V;
    constexpr int kN = Vec16<TIn>::N;
    constexpr int kMaxPer = (kBT * NMAX / kN + kBwdThreads - 1) / kBwdThreads;
    const int nvec = kBT * n / kN;
    V buf[kMaxPer];
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        const int idx = tid + kBwdThreads * i;
        buf[i] = V{};
        if (idx < nvec && r0 + (idx * kN) / n < nrows_total)
            buf[i] = reinterpret_cast<const V*>(src + static_cast<int64_t>(r0) * n)[idx];
    }
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        const int idx = tid + kBwdThreads * i;
        if (idx < nvec) {
            const int e = idx * kN;
            *reinterpret_cast<V*>(dst + (e / n) * pitch + e % n) = buf[i];
        }
    }
}

template <typename TIn, int NK, int NV>   // DQK = 64 NK, DV = 64 NV
__global__ void __launch_bounds__(kBwdThreads) bwd_row_mfma_kernel(BwdArgs A) {
    extern __shared__ float sm[];
    constexpr int DQK = 64 * NK, DV = 64 * NV;
    const int T = A.T;
    constexpr int KP = DQK + lds_pad<TIn>(), VP = DV + lds_pad<TIn>();
    TIn* Ks = reinterpret_cast<TIn*>(sm);                // [kBT][KP]
    TIn* Vs = Ks + kBT * KP;                             // [kBT][VP]
    float* Pr = reinterpret_cast<float*>(Vs + kBT * VP); // [4 waves][kBT][kBT] partial logits
    float* Op = Pr + 4 * kBT * kBT;      // [kBT][kTP] operand tile (A~ or W), rows t
    float* red = Op + kBT * kTP;         // [4][kBT][kBT] row partial sums
    float* rowv = red + 4 * kBT * kBT;   // [kBT][4] per row: M, m, dD
    const int ntile = (T + kBT - 1) / kBT;
    const int64_t seq = blockIdx.x / ntile;
    const int t0 = (blockIdx.x % ntile) * kBT;
    MLSTM_CHECK(t0 < T && DQK % 16 == 0 && DV % 16 == 0, kDbgParallelBwd);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, g = lane >> 4;
    const int pr = tid / kBT, pc = tid % kBT;
    const TIn* q = static_cast<const TIn*>(A.q) + seq * T * DQK;
    const TIn* k = static_cast<const TIn*>(A.k) + seq * T * DQK;
    const TIn* v = static_cast<const TIn*>(A.v) + seq * T * DV;
    float* wsq = A.ws + seq * ws_floats(T, DV);
    const float* xw = wsq;
    const float* Mw = wsq + T;
    const float* mw = wsq + 2 * T;
    float* dDw = wsq + 3 * T;
    float* Pw = wsq + 4 * T;
    float* dNw = wsq + dn_off(T);
    const float qscale = rsqrtf(static_cast<float>(DQK));
    constexpr int nvt = NV, nkt = NK;   // 16-column output tiles per wave
    const int vc0 = wave * (DV / 4), kc0 = wave * (DQK / 4);

    // this wave's quarter of the q^ rows, as the A operand of the logits (lane: row l16, k 4 kk + g)
    constexpr int kq = DQK / 4;
    float qreg[(4 * NK)];
#pragma unroll
    for (int kk = 0; kk < (4 * NK); ++kk)
        qreg[kk] = (kk < kq / 4 && t0 + l16 < T)
                       ? io<TIn>::load(q, static_cast<int64_t>(t0 + l16) * DQK + wave * kq + 4 * kk + g) * qscale
                       : 0.0f;
    if (tid < kBT) {
        const int t = t0 + tid;
        rowv[4 * tid + 0] = t < T ? Mw[t] : 0.0f;
        rowv[4 * tid + 1] = t < T ? mw[t] : 0.0f;
    }
    f32x4_t accN[NV];
#pragma unroll
    for (int c = 0; c < NV; ++c) accN[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float accD = 0.0f;   // this thread's (t, s) column of A~, summed over s tiles
    const int t_pair = t0 + pr;
    const int last_tile = t0 / kBT;

    for (int st = 0; st <= last_tile; ++st) {
        const int s0 = st * kBT;
        __syncthreads();
        stage_raw<TIn, DQK>(Ks, KP, k, s0, T, DQK, tid);
        stage_raw<TIn, DV>(Vs, VP, v, s0, T, DV, tid);
        __syncthreads();
        f32x4_t part = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < (4 * NK); ++kk)
            if (kk < kq / 4) part = mfma4(qreg[kk], lds_ld(Ks, l16 * KP + wave * kq + 4 * kk + g), part);
#pragma unroll
        for (int j = 0; j < 4; ++j) Pr[(wave * kBT + 4 * g + j) * kBT + l16] = part[j];
        __syncthreads();
        {
            const int s = s0 + pc;
            float a = 0.0f;
            if (s <= t_pair && t_pair < T) {
                const float sv = Pr[pr * kBT + pc] + Pr[(kBT + pr) * kBT + pc] + Pr[(2 * kBT + pr) * kBT + pc] +
                                 Pr[(3 * kBT + pr) * kBT + pc];
                a = expf(xw[s] - rowv[4 * pr]) * sv;
            }
            Op[pr * kTP + pc] = a;
            accD += a;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const float a = Op[l16 * kTP + 4 * kk + g];
#pragma unroll
            for (int c = 0; c < NV; ++c)
                if (c < nvt) accN[c] = mfma4(a, lds_ld(Vs, (4 * kk + g) * VP + vc0 + 16 * c + l16), accN[c]);
        }
    }
    // D~ per row, then dN~, dD~ and P
    red[pr * kBT + pc] = accD;
    __syncthreads();
    if (tid < kBT) {
        float d = 0.0f;
        for (int j = 0; j < kBT; ++j) d += red[tid * kBT + j];
        rowv[4 * tid + 3] = d;
    }
    __syncthreads();
    float part_hh[4] = {0.f, 0.f, 0.f, 0.f}, part_nn[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = 4 * g + j, t = t0 + r;
        const float Dt = rowv[4 * r + 3];
        const float den = fmaxf(fabsf(Dt), expf(-rowv[4 * r + 1]));
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            if (c < nvt) {
                const int col = vc0 + 16 * c + l16;
                const float gh = t < T ? A.dh[(seq * T + t) * DV + col] : 0.0f;
                const float nv = accN[c][j];
                const float dn = gh / den;
                part_hh[j] += gh * (nv / den);
                part_nn[j] += dn * nv;
                if (t < T) dNw[static_cast<int64_t>(t) * DV + col] = dn;
            }
        }
    }
    // row sums over the 16 lanes of a row group and the four waves
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        red[(wave * kBT + 4 * g + j) * kBT + l16] = part_hh[j];
    }
    __syncthreads();
    if (tid < kBT) {
        float sdh = 0.0f;
        for (int w = 0; w < 4; ++w)
            for (int j = 0; j < kBT; ++j) sdh += red[(w * kBT + tid) * kBT + j];
        const float Dt = rowv[4 * tid + 3];
        const float fl = expf(-rowv[4 * tid + 1]);
        const float den = fmaxf(fabsf(Dt), fl);
        rowv[4 * tid + 2] = (fabsf(Dt) > fl) ? -sdh / den * (Dt > 0.0f ? 1.0f : -1.0f) : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) red[(wave * kBT + 4 * g + j) * kBT + l16] = part_nn[j];
    __syncthreads();
    if (tid < kBT && t0 + tid < T) {
        float sdn = 0.0f;
        for (int w = 0; w < 4; ++w)
            for (int j = 0; j < kBT; ++j) sdn += red[(w * kBT + tid) * kBT + j];
        const float dD = rowv[4 * tid + 2];
        dDw[t0 + tid] = dD;
        Pw[t0 + tid] = sdn + dD * rowv[4 * tid + 3];
    }

    // dN~ rows into registers as the A operand of U = dN~ V^T (lane: row l16, d = this wave's
    // quarter, 4 kk + g), read back from the workspace: the wave stored exactly these columns
    // above, and the barriers since then order the stores before the loads
    constexpr int dq4 = DV / 4;
    __syncthreads();
    float dnreg[(4 * NV)];
#pragma unroll
    for (int kk = 0; kk < (4 * NV); ++kk)
        dnreg[kk] = (kk < dq4 / 4 && t0 + l16 < T)
                        ? dNw[static_cast<int64_t>(t0 + l16) * DV + wave * dq4 + 4 * kk + g] : 0.0f;

    // sweep 2: dq
    f32x4_t accQ[NK];
#pragma unroll
    for (int c = 0; c < NK; ++c) accQ[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int st = 0; st <= last_tile; ++st) {
        const int s0 = st * kBT;
        __syncthreads();
        stage_raw<TIn, DQK>(Ks, KP, k, s0, T, DQK, tid);
        stage_raw<TIn, DV>(Vs, VP, v, s0, T, DV, tid);
        __syncthreads();
        f32x4_t part = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < (4 * NV); ++kk)
            if (kk < dq4 / 4) part = mfma4(dnreg[kk], lds_ld(Vs, l16 * VP + wave * dq4 + 4 * kk + g), part);
#pragma unroll
        for (int j = 0; j < 4; ++j) Pr[(wave * kBT + 4 * g + j) * kBT + l16] = part[j];
        __syncthreads();
        {
            const int s = s0 + pc;
            float w = 0.0f;
            if (s <= t_pair && t_pair < T) {
                const float u = Pr[pr * kBT + pc] + Pr[(kBT + pr) * kBT + pc] + Pr[(2 * kBT + pr) * kBT + pc] +
                                Pr[(3 * kBT + pr) * kBT + pc];
                w = (u + rowv[4 * pr + 2]) * expf(xw[s] - rowv[4 * pr]);
            }
            Op[pr * kTP + pc] = w;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const float a = Op[l16 * kTP + 4 * kk + g];
#pragma unroll
            for (int c = 0; c < NK; ++c)
                if (c < nkt) accQ[c] = mfma4(a, lds_ld(Ks, (4 * kk + g) * KP + kc0 + 16 * c + l16), accQ[c]);
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int t = t0 + 4 * g + j;
        if (t < T) {
#pragma unroll
            for (int c = 0; c < NK; ++c)
                if (c < nkt) A.dq[(seq * T + t) * DQK + kc0 + 16 * c + l16] = accQ[c][j] * qscale;
        }
    }
}

// With bf16 inputs three workgroups fit a CU's LDS; the register budget is capped to match (a few
// registers spill, and it is still faster than two workgroups).  fp32 tiles allow two.
template <typename TIn> constexpr int col_waves() { return sizeof(TIn) == 2 ? 3 : 2; }
template <typename TIn, int NK, int NV>   // DQK = 64 NK, DV = 64 NV
__global__ void __launch_bounds__(kBwdThreads) __attribute__((amdgpu_waves_per_eu(col_waves<TIn>())))
bwd_col_mfma_kernel(BwdArgs A) {
    extern __shared__ float sm[];
    constexpr int DQK = 64 * NK, DV = 64 * NV;
    const int T = A.T;
    constexpr int KP = DQK + lds_pad<TIn>(), VP = DV + 4;
    TIn* Qs = reinterpret_cast<TIn*>(sm);                // [kBT][KP] a tile of q (unscaled)
    float* dN = reinterpret_cast<float*>(Qs + kBT * KP); // [kBT][VP] a tile of dN~
    float* Ps = dN + kBT * VP;           // [4][kBT][kBT] partial S
    float* Pu = Ps + 4 * kBT * kBT;      // [4][kBT][kBT] partial U
    float* Wt = Pu + 4 * kBT * kBT;      // [kBT][kTP] W^T (rows s)
    float* At = Wt + kBT * kTP;          // [kBT][kTP] A~^T (rows s)
    float* red = At + kBT * kTP;         // [kBT][kBT]
    float* rowv = red + kBT * kBT;       // [kBT][2] per row t of the t tile: M, dD
    const int ntile = (T + kBT - 1) / kBT;
    const int64_t seq = blockIdx.x / ntile;
    const int s0 = (blockIdx.x % ntile) * kBT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, g = lane >> 4;
    const int pr = tid / kBT, pc = tid % kBT;   // pair (t row pr, s column pc)
    const TIn* q = static_cast<const TIn*>(A.q) + seq * T * DQK;
    const TIn* k = static_cast<const TIn*>(A.k) + seq * T * DQK;
    const TIn* v = static_cast<const TIn*>(A.v) + seq * T * DV;
    const float* wsq = A.ws + seq * ws_floats(T, DV);
    const float* xw = wsq;
    const float* Mw = wsq + T;
    const float* dDw = wsq + 3 * T;
    const float* dNw = wsq + dn_off(T);
    const float qscale = rsqrtf(static_cast<float>(DQK));
    constexpr int nvt = NV, nkt = NK;
    const int vc0 = wave * (DV / 4), kc0 = wave * (DQK / 4);

    // this tile's k and v rows, as the B operands of S and U (lane: column s = l16, the wave's
    // quarter of the contraction, 4 kk + g)
    constexpr int kq = DQK / 4, dq4 = DV / 4;
    float kreg[(4 * NK)], vreg[(4 * NV)];
#pragma unroll
    for (int kk = 0; kk < (4 * NK); ++kk)
        kreg[kk] = (kk < kq / 4 && s0 + l16 < T)
                       ? io<TIn>::load(k, static_cast<int64_t>(s0 + l16) * DQK + wave * kq + 4 * kk + g) : 0.0f;
#pragma unroll
    for (int kk = 0; kk < (4 * NV); ++kk)
        vreg[kk] = (kk < dq4 / 4 && s0 + l16 < T)
                       ? io<TIn>::load(v, static_cast<int64_t>(s0 + l16) * DV + wave * dq4 + 4 * kk + g) : 0.0f;
    f32x4_t accK[NK], accV[NV];
#pragma unroll
    for (int c = 0; c < NK; ++c) accK[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NV; ++c) accV[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float accI = 0.0f;   // this thread's (t, s) entry of G, summed over t tiles
    for (int tt = s0 / kBT; tt < ntile; ++tt) {
        const int t0 = tt * kBT;
        __syncthreads();
        stage_raw<TIn, DQK>(Qs, KP, q, t0, T, DQK, tid);
        stage_rows_f32<DV>(dN, VP, dNw, t0, T, DV, tid);
        if (tid < kBT) {
            const int t = t0 + tid;
            rowv[2 * tid + 0] = t < T ? Mw[t] : 0.0f;
            rowv[2 * tid + 1] = t < T ? dDw[t] : 0.0f;
        }
        __syncthreads();
        f32x4_t ps = f32x4_t{0.f, 0.f, 0.f, 0.f}, pu = f32x4_t{0.f, 0.f, 0.f, 0.f};   // S[t][s], U[t][s]
#pragma unroll
        for (int kk = 0; kk < (4 * NK); ++kk)
            if (kk < kq / 4) ps = mfma4(lds_ld(Qs, l16 * KP + wave * kq + 4 * kk + g), kreg[kk], ps);
#pragma unroll
        for (int kk = 0; kk < (4 * NV); ++kk)
            if (kk < dq4 / 4) pu = mfma4(dN[l16 * VP + wave * dq4 + 4 * kk + g], vreg[kk], pu);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            Ps[(wave * kBT + 4 * g + j) * kBT + l16] = ps[j] * qscale;
            Pu[(wave * kBT + 4 * g + j) * kBT + l16] = pu[j];
        }
        __syncthreads();
        {
            const int t = t0 + pr, s = s0 + pc;
            float w = 0.0f, a = 0.0f;
            if (s <= t && t < T && s < T) {
                float sv = 0.0f, u = 0.0f;
#pragma unroll
                for (int w4 = 0; w4 < 4; ++w4) {
                    sv += Ps[(w4 * kBT + pr) * kBT + pc];
                    u += Pu[(w4 * kBT + pr) * kBT + pc];
                }
                const float F = expf(xw[s] - rowv[2 * pr]);
                w = (u + rowv[2 * pr + 1]) * F;
                a = F * sv;
                accI += w * sv;
            }
            Wt[pc * kTP + pr] = w;
            At[pc * kTP + pr] = a;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const float aw = Wt[l16 * kTP + 4 * kk + g];
            const float aa = At[l16 * kTP + 4 * kk + g];
#pragma unroll
            for (int c = 0; c < NK; ++c)
                if (c < nkt) accK[c] = mfma4(aw, lds_ld(Qs, (4 * kk + g) * KP + kc0 + 16 * c + l16), accK[c]);
#pragma unroll
            for (int c = 0; c < NV; ++c)
                if (c < nvt) accV[c] = mfma4(aa, dN[(4 * kk + g) * VP + vc0 + 16 * c + l16], accV[c]);
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int s = s0 + 4 * g + j;
        if (s < T) {
#pragma unroll
            for (int c = 0; c < NK; ++c)
                if (c < nkt) A.dk[(seq * T + s) * DQK + kc0 + 16 * c + l16] = accK[c][j] * qscale;
#pragma unroll
            for (int c = 0; c < NV; ++c)
                if (c < nvt) A.dv[(seq * T + s) * DV + vc0 + 16 * c + l16] = accV[c][j];
        }
    }
    red[pr * kBT + pc] = accI;
    __syncthreads();
    if (tid < kBT && s0 + tid < T) {
        float d = 0.0f;
        for (int r = 0; r < kBT; ++r) d += red[r * kBT + tid];
        A.dipre[seq * T + s0 + tid] = d;
    }
}

// ---- forget pass -------------------------------------------------------------------------------
// one wave per sequence, from the last token backwards, 64 tokens per step (lane 0 the latest)
__global__ void bwd_forget_kernel(BwdArgs A, int S) {
    const int s = blockIdx.x;
    const int lane = threadIdx.x;
    const int T = A.T;
    const float* Pw = A.ws + s * ws_floats(T, A.DV) + 4 * T;
    const float* di = A.dipre + static_cast<int64_t>(s) * T;
    const float* fb = A.fpre + static_cast<int64_t>(s) * T;
    float* df = A.dfpre + static_cast<int64_t>(s) * T;
    float carry = 0.0f;
    for (int eb = T - 1; eb >= 0; eb -= 64 * kScanBatch) {
        float pv[kScanBatch], fv[kScanBatch];
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u) {
            const int j = eb - 64 * u - lane;
            pv[u] = j >= 0 ? Pw[j] - di[j] : 0.0f;
            fv[u] = j >= 0 ? fb[j] : 0.0f;
        }
        float ls[kScanBatch], lt[kScanBatch];   // independent scans first, then the carries in order
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u) {
            ls[u] = wave_scan_sum(pv[u], lane);
            lt[u] = __shfl(ls[u], 63, 64);
        }
#pragma unroll
        for (int u = 0; u < kScanBatch; ++u) {
            const int j = eb - 64 * u - lane;
            if (j >= 0) df[j] = (carry + ls[u]) / (1.0f + expf(fv[u]));   // sigmoid(-f~)
            carry += lt[u];
        }
    }
}

template <typename TIn>
size_t row_mfma_lds(int DQK, int DV) {
    return sizeof(TIn) * (kBT * (DQK + lds_pad<TIn>()) + kBT * (DV + lds_pad<TIn>())) +
           sizeof(float) * (4 * kBT * kBT + kBT * kTP + 4 * kBT * kBT + 4 * kBT);
}
template <typename TIn>
size_t col_mfma_lds(int DQK, int DV) {
    return sizeof(TIn) * kBT * (DQK + lds_pad<TIn>()) +
           sizeof(float) * (kBT * (DV + 4) + 8 * kBT * kBT + 2 * kBT * kTP + kBT * kBT + 2 * kBT);
}
size_t row_lds(int DQK, int DV) {
    return sizeof(float) * (2 * kBT * (DQK + 1) + 2 * kBT * (DV + 1) + 2 * kBT * kBT + 4 * kBT);
}
size_t col_lds(int DQK, int DV) {
    return sizeof(float) * (2 * kBT * (DQK + 1) + 2 * kBT * (DV + 1) + 3 * kBT * kBT + 2 * kBT);
}

// The MFMA passes for one (DQK, DV) = (64 NK, 64 NV); their dynamic LDS limit is raised once per device.
template <typename TIn, int NK, int NV>
hipError_t launch_mfma_passes(const BwdArgs& a, dim3 tiles, hipStream_t stream) {
    static std::atomic<uint64_t> raised_row{0}, raised_col{0};
    const size_t lr = row_mfma_lds<TIn>(64 * NK, 64 * NV), lc = col_mfma_lds<TIn>(64 * NK, 64 * NV);
    hipError_t e = raise_dynamic_lds(reinterpret_cast<const void*>(bwd_row_mfma_kernel<TIn, NK, NV>), lr, raised_row);
    if (e == hipSuccess)
        e = raise_dynamic_lds(reinterpret_cast<const void*>(bwd_col_mfma_kernel<TIn, NK, NV>), lc, raised_col);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((bwd_row_mfma_kernel<TIn, NK, NV>), tiles, dim3(kBwdThreads), lr, stream, a);
    hipLaunchKernelGGL((bwd_col_mfma_kernel<TIn, NK, NV>), tiles, dim3(kBwdThreads), lc, stream, a);
    return hipSuccess;
}

// head shapes with MFMA passes: the xLSTM-7B head and three smaller ones
bool bwd_mfma_shape(int DQK, int DV) {
    return (DQK == 256 && DV == 512) || (DQK == 64 && DV == 64) || (DQK == 64 && DV == 128) ||
           (DQK == 128 && DV == 192);
}

template <typename TIn>
hipError_t launch_typed(const BwdArgs& a, int S, hipStream_t stream) {
    static std::atomic<uint64_t> raised_row{0}, raised_col{0};
    {
        hipError_t e = raise_dynamic_lds(reinterpret_cast<const void*>(bwd_row_kernel<TIn>), row_lds(kMaxDQK, kMaxDV),
                                         raised_row);
        if (e == hipSuccess)
            e = raise_dynamic_lds(reinterpret_cast<const void*>(bwd_col_kernel<TIn>), col_lds(kMaxDQK, kMaxDV),
                                  raised_col);
        if (e != hipSuccess) return e;
    }
    const int ntile = (a.T + kBT - 1) / kBT;
    const dim3 tiles(static_cast<unsigned>(static_cast<int64_t>(S) * ntile));
    const dim3 seqs(static_cast<unsigned>(S));   // the scans: one wave per sequence
    hipLaunchKernelGGL(bwd_gate_kernel, seqs, dim3(64), 0, stream, a, S);
    hipError_t e = hipSuccess;
    if (a.DQK == 256 && a.DV == 512) e = launch_mfma_passes<TIn, 4, 8>(a, tiles, stream);
    else if (a.DQK == 64 && a.DV == 64) e = launch_mfma_passes<TIn, 1, 1>(a, tiles, stream);
    else if (a.DQK == 64 && a.DV == 128) e = launch_mfma_passes<TIn, 1, 2>(a, tiles, stream);
    else if (a.DQK == 128 && a.DV == 192) e = launch_mfma_passes<TIn, 2, 3>(a, tiles, stream);
    else {
        hipLaunchKernelGGL(bwd_row_kernel<TIn>, tiles, dim3(kBwdThreads), row_lds(a.DQK, a.DV), stream, a);
        hipLaunchKernelGGL(bwd_col_kernel<TIn>, tiles, dim3(kBwdThreads), col_lds(a.DQK, a.DV), stream, a);
    }
    if (e != hipSuccess) return e;
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

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_parallel_bwd)
#endif

}  // namespace mlstm
