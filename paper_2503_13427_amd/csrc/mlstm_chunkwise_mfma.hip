// Chunkwise-parallel mLSTM forward on bf16 MFMA for the xLSTM 7B head shape
// (DQK = 256, DV = 512; Sec. 3.1 sets d_qk = d_hv / 2 and d_hv = 512), chunk
// size L in {64, 128}.
//
// Math.  The chunkwise form of Sec. 2 ("Training Mode") with the sub-steps of
// App. D.1.  Per chunk, with the entry state (C, n, m_prev), in-chunk prefix
// sums b of logsig(f~), x = i~ - b, p_tau = max_{sig<=tau} x_sig and
// M_tau = max(m_prev, p_tau) (so the max state of Eq. 2 is m_tau = b_tau + M_tau):
//
//   S~^T[sig][tau] = (K Q^T)[sig][tau] / sqrt(DQK) * exp(x_sig - M_tau)   (sig <= tau, else 0)
//   N^T            = exp(m_prev - M_tau)/sqrt(DQK) * (C^T Q^T)  +  V^T S~^T
//   den_tau        = exp(m_prev - M_tau)/sqrt(DQK) * (Q n)_tau  +  rowsum_tau(S~)
//   h_tau          = N^T[:, tau] / max(|den_tau|, exp(-(b_tau + M_tau)))
//   C <- exp(m_prev - M_L) C + (w K)^T V,  n <- exp(m_prev - M_L) n + K^T w,
//   w_tau = exp(x_tau - M_L),  m_next = b_L + M_L.
// Every exponent is a difference against M and is <= 0 by construction.
//
// Products and their MFMA mapping (gfx950 bf16 MFMA, fp32 accumulate):
//   (i)   S^T = K Q^T             16x16x32: A = K rows, B = Q rows (both d-contiguous)
//   (ii)  N^T += V^T S~^T         32x32x16: A = V^T (sigma-contiguous), B = S~ rows
//   (iii) N^T += C^T Q^T          32x32x16: A = C straight from the accumulators of
//                                 (iv), converted to bf16 in registers, B = Q rows
//   (iv)  C += (wK)^T V           32x32x16: A = (wK)^T, B = V^T (both tau-contiguous)
// (iii) consumes C in the accumulator layout of (iv): the contraction index d is
// permuted consistently in both operands, so no LDS round trip is needed.  The
// outputs come out transposed (rows v, columns tau), so each lane holds runs of
// four consecutive v of one h row and stores 8 bytes at a time.
//
// Work decomposition.  One workgroup of 4 waves owns one (sequence, 128-column
// dv tile, segment) and walks the segment's chunks in order.  Wave w owns the
// 256 x 32 fp32 slice C[:, 32w:32w+32] of the matrix memory in its MFMA
// accumulators for the whole segment (128 registers per lane); n lives in LDS.
// Within a chunk, Q and K are staged in four 64-wide d blocks; the next block
// (and the next chunk's V and gates) is prefetched into registers while the
// current block is multiplied.  K^T and V^T are transposed in registers on the
// way into LDS.  The four dv tiles of a (sequence, segment) are dispatched
// consecutively onto the same XCD so their shared Q/K reads hit one L2.
//
// Segment-parallel schedule (optional workspace).  With G segments per
// sequence: (1) the LOCAL variant computes each of the first G-1 segments' state
// from an empty state (C = 0, n = 0, m = -inf) -- gates, (wK)^T V and n only;
// (2) a combine kernel scans those local states into each segment's entry state,
// m_in' = max(gsum + m_in, m_loc), C_in' = e^{gsum + m_in - m_in'} C_in + e^{m_loc - m_in'} C_loc;
// (3) the FULL variant runs every segment from its entry state.
#include "device_common.h"
#include "launch.h"

namespace mlstm {
namespace {

constexpr int kDQK = 256;
constexpr int kDV = 512;
constexpr int kDVT = 128;             // dv columns per workgroup
constexpr int kNTile = kDV / kDVT;    // 4 dv tiles per sequence
constexpr int kDB = 64;               // d block staged per step
constexpr int kNDB = kDQK / kDB;      // 4 d blocks
constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kQScale = 0.0625f;    // 1 / sqrt(256), exact

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4_t mfma16(u32x4_t a, u32x4_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_t mfma32(u32x4_t a, u32x4_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                   c, 0, 0, 0);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 pair, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ float lo_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f32(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t lo16(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ __forceinline__ uint32_t hi16(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int L>
struct Smem {
    static constexpr int QP = kDB + 8;   // row pitch (elements) of the d-contiguous Q/K block tiles
    static constexpr int TP = L + 8;     // row pitch of the tau-contiguous tiles
    static constexpr int NB = L / 16;    // 16-wide blocks along the chunk
    uint16_t Qb[L * QP];                 // Q[tau][d]  (current d block)
    uint16_t Kb[L * QP];                 // K[tau][d]
    uint16_t Ktb[kDB * TP];              // (w K)^T[d][tau]
    uint16_t Vt[kDVT * TP];              // V^T[v][tau]  (this workgroup's 128 columns)
    uint16_t St[L * TP];                 // S~[tau][sig]
    float n[2][kDQK];                    // normaliser, double-buffered across chunks
    float x2[L];                         // (i~ - b) * log2 e
    float M2[L];                         // M * log2 e
    float inter[L];                      // exp(m_prev - M) / sqrt(DQK)
    float floorv[L];                     // exp(-(b + M))
    float w[L];                          // key weights exp(x - M_L)
    float dq[L];                         // Q n_{k-1} (unscaled q)
    float hinv[L];                       // 1 / max(|den|, floor)
    float rs[NB][L];                     // row sums of S~ per 16-wide sigma block
    float scal[4];                       // [0] decay, [1] m_next, [2] gsum (log forget total)
};

// Per-thread staging registers.
template <int L>
struct QKRegs {
    static constexpr int NQ = (L * kDB / 8) / kThreads;   // 16-byte Q chunks per thread
    static constexpr int NK = (L / 4) * (kDB / 4) / kThreads;   // 4x4 K blocks per thread
    u32x4_t q[NQ];
    u32x2_t k[NK][4];
};
template <int L>
struct VRegs {
    static constexpr int NV = (L / 8) * (kDVT / 4) / kThreads;   // 8x4 V blocks per thread
    u32x2_t v[NV][8];
    float ig, fg, ig2, fg2;   // gates (wave 0; two per lane when L == 128)
};

// Buffer resources (SGPRs) for one sequence's inputs: loads then need one 32-bit
// VGPR offset per staging item plus immediate offsets, instead of a 64-bit
// address per load.  Out-of-range buffer reads return zero.
constexpr int kRsrcWord3 = 0x00020000;

struct SeqRsrc {
    __amdgpu_buffer_rsrc_t q, k, v, ig, fg;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0), static_cast<int>(bytes),
                                             kRsrcWord3);
}
__device__ __forceinline__ u32x4_t bload128(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ u32x2_t bload64(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}
__device__ __forceinline__ float bloadf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// q/k rows are 512 bytes, v rows 1024 bytes; offsets below are in bytes.
template <int L, bool FULL>
__device__ __forceinline__ void load_qk(QKRegs<L>& r, const SeqRsrc& R, int t0, int p, int tid) {
    const uint32_t soff = static_cast<uint32_t>(t0) * (kDQK * 2) + p * (kDB * 2);
    if constexpr (FULL) {
#pragma unroll
        for (int i = 0; i < QKRegs<L>::NQ; ++i) {
            const int item = tid + i * kThreads;
            const int tau = item >> 3, c = item & 7;
            r.q[i] = bload128(R.q, tau * (kDQK * 2) + 16 * c, soff);
        }
    }
#pragma unroll
    for (int i = 0; i < QKRegs<L>::NK; ++i) {
        const int item = tid + i * kThreads;
        const int dg = item & 15, tg = item >> 4;
        const uint32_t voff = (4 * tg) * (kDQK * 2) + 8 * dg;
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) r.k[i][r4] = bload64(R.k, voff + r4 * (kDQK * 2), soff);
    }
}

template <int L>
__device__ __forceinline__ void load_v(VRegs<L>& r, const SeqRsrc& R, int t0, int v0, int tid) {
    const uint32_t soff = static_cast<uint32_t>(t0) * (kDV * 2) + v0 * 2;
#pragma unroll
    for (int i = 0; i < VRegs<L>::NV; ++i) {
        const int item = tid + i * kThreads;
        const int vg = item & 31, tg = item >> 5;
        const uint32_t voff = (8 * tg) * (kDV * 2) + 8 * vg;
#pragma unroll
        for (int r8 = 0; r8 < 8; ++r8) r.v[i][r8] = bload64(R.v, voff + r8 * (kDV * 2), soff);
    }
    if (tid < 64) {
        const uint32_t goff = static_cast<uint32_t>(t0) * 4;
        r.ig = bloadf(R.ig, 4 * tid, goff);
        r.fg = bloadf(R.fg, 4 * tid, goff);
        if constexpr (L == 128) {
            r.ig2 = bloadf(R.ig, 4 * tid + 256, goff);
            r.fg2 = bloadf(R.fg, 4 * tid + 256, goff);
        }
    }
}

template <int L, bool FULL>
__device__ __forceinline__ void store_qk(Smem<L>& S, const QKRegs<L>& r, int tid) {
    constexpr int QP = Smem<L>::QP, TP = Smem<L>::TP;
    if constexpr (FULL) {
#pragma unroll
        for (int i = 0; i < QKRegs<L>::NQ; ++i) {
            const int item = tid + i * kThreads;
            const int tau = item >> 3, c = item & 7;
            *reinterpret_cast<u32x4_t*>(&S.Qb[tau * QP + 8 * c]) = r.q[i];
        }
    }
#pragma unroll
    for (int i = 0; i < QKRegs<L>::NK; ++i) {
        const int item = tid + i * kThreads;
        const int dg = item & 15, tg = item >> 4;
        float wv[4];
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            *reinterpret_cast<u32x2_t*>(&S.Kb[(4 * tg + r4) * QP + 4 * dg]) = r.k[i][r4];
            wv[r4] = S.w[4 * tg + r4];
        }
        // (w K)^T for d = 4dg..4dg+3, tau = 4tg..4tg+3
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float kv[4];
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const uint32_t word = r.k[i][r4][c >> 1];
                kv[r4] = ((c & 1) ? hi_f32(word) : lo_f32(word)) * wv[r4];
            }
            u32x2_t o;
            o[0] = pack_bf16x2(kv[0], kv[1]);
            o[1] = pack_bf16x2(kv[2], kv[3]);
            *reinterpret_cast<u32x2_t*>(&S.Ktb[(4 * dg + c) * TP + 4 * tg]) = o;
        }
    }
}

template <int L>
__device__ __forceinline__ void store_v(Smem<L>& S, const VRegs<L>& r, int tid) {
    constexpr int TP = Smem<L>::TP;
#pragma unroll
    for (int i = 0; i < VRegs<L>::NV; ++i) {
        const int item = tid + i * kThreads;
        const int vg = item & 31, tg = item >> 5;
        // 8 rows (tau) x 4 columns (v) -> 4 rows of V^T with 8 consecutive tau
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            u32x4_t o;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const uint32_t a = r.v[i][2 * m][c >> 1], b = r.v[i][2 * m + 1][c >> 1];
                o[m] = (c & 1) ? hi16(a, b) : lo16(a, b);
            }
            *reinterpret_cast<u32x4_t*>(&S.Vt[(4 * vg + c) * TP + 8 * tg]) = o;
        }
    }
}

// Inclusive wave-wide scans over 64 lanes.
__device__ __forceinline__ float wave_incl_sum(float x, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    return x;
}
__device__ __forceinline__ float wave_incl_max(float x, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float y = __shfl_up(x, o, 64);
        if (lane >= o) x = fmaxf(x, y);
    }
    return x;
}

// Gate phase (wave 0): chunkwise gates, max state and all per-row scales.
template <int L>
__device__ __forceinline__ void gate_phase(Smem<L>& S, const VRegs<L>& r, float m_prev, int lane) {
    float a = logsigmoid(r.fg);
    float b = wave_incl_sum(a, lane);
    float x = r.ig - b;
    float p = wave_incl_max(x, lane);
    float b2 = 0.f, x2 = 0.f, p2 = 0.f;
    if constexpr (L == 128) {
        const float btot = __shfl(b, 63, 64);
        const float ptot = __shfl(p, 63, 64);
        b2 = btot + wave_incl_sum(logsigmoid(r.fg2), lane);
        x2 = r.ig2 - b2;
        p2 = fmaxf(ptot, wave_incl_max(x2, lane));
    }
    const float pL = (L == 128) ? __shfl(p2, 63, 64) : __shfl(p, 63, 64);
    const float bL = (L == 128) ? __shfl(b2, 63, 64) : __shfl(b, 63, 64);
    const float ML = fmaxf(m_prev, pL);
    // An empty state (m = -inf, only in the local-state pass) contributes nothing; the guards
    // keep -inf - -inf out of the exponentials when a chunk also writes nothing (all i~ = -inf).
    auto emit = [&](int tau, float bb, float xx, float pp) {
        const float M = fmaxf(m_prev, pp);
        S.x2[tau] = xx * kLog2e;
        S.M2[tau] = M * kLog2e;
        S.inter[tau] = (M == -INFINITY) ? 0.0f : expf(m_prev - M) * kQScale;
        S.floorv[tau] = expf(-(bb + M));
        S.w[tau] = (xx == -INFINITY) ? 0.0f : expf(xx - ML);
    };
    emit(lane, b, x, p);
    if constexpr (L == 128) emit(64 + lane, b2, x2, p2);
    if (lane == 0) {
        S.scal[0] = (ML == -INFINITY) ? 0.0f : expf(m_prev - ML);
        S.scal[1] = bL + ML;
        S.scal[2] += bL;
    }
}

// XCD-aware block order: the hardware deals consecutive workgroups round-robin
// to the 8 XCDs; renumber so that consecutive work items (the four dv tiles of a
// sequence/segment) run on the same XCD.
__device__ __forceinline__ int work_index() {
    const int nb = gridDim.x, b = blockIdx.x;
    if (nb % 8) return b;
    return (b % 8) * (nb / 8) + b / 8;
}

struct ChunkKernelArgs {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const float* ipre;
    const float* fpre;
    const float* C0;   // entry state of segment 0 (NULL: zero state, m = 0)
    const float* n0;
    const float* m0;
    float* ws;         // segment slots (NULL when G == 1)
    int T;
    int G;             // segments per sequence
    int seg_chunks;    // chunks per segment (last may be shorter)
    uint16_t* h;
    float* CT;
    float* nT;
    float* mT;
};

// workspace slot of (sequence s, segment g): C [DQK*DV], n [DQK], then m_loc, gsum, m_in, pad
constexpr int64_t kSlotFloats = static_cast<int64_t>(kDQK) * kDV + kDQK + 4;

template <int L, bool FULL>
__global__ void __launch_bounds__(kThreads, 1) chunk_mfma_kernel(ChunkKernelArgs A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    Smem<L>& S = *reinterpret_cast<Smem<L>*>(smem_raw);
    constexpr int QP = Smem<L>::QP, TP = Smem<L>::TP, NB = Smem<L>::NB;
    constexpr int NT_S = NB * (NB + 1) / 2;          // causal 16x16 tiles of S^T
    constexpr int MAXT = (NT_S + kWaves - 1) / kWaves;
    constexpr int NTT = L / 32;                       // 32-wide tau tiles

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kg = lane >> 5;   // 32x32 k group
    const int l32 = lane & 31;
    const int g16 = lane >> 4;  // 16x16 k group
    const int l16 = lane & 15;

    const int wi = work_index();
    const int tile = wi % kNTile;
    const int sg = wi / kNTile;
    const int G_run = FULL ? A.G : A.G - 1;
    const int g = sg % G_run;
    const int s = sg / G_run;
    const int v0 = tile * kDVT;
    const int nc_total = A.T / L;
    const int c_begin = g * A.seg_chunks;
    const int c_end = min(nc_total, c_begin + A.seg_chunks);

    SeqRsrc P;
    P.q = make_rsrc(A.q + static_cast<int64_t>(s) * A.T * kDQK, static_cast<uint32_t>(A.T) * kDQK * 2);
    P.k = make_rsrc(A.k + static_cast<int64_t>(s) * A.T * kDQK, static_cast<uint32_t>(A.T) * kDQK * 2);
    P.v = make_rsrc(A.v + static_cast<int64_t>(s) * A.T * kDV, static_cast<uint32_t>(A.T) * kDV * 2);
    P.ig = make_rsrc(A.ipre + static_cast<int64_t>(s) * A.T, static_cast<uint32_t>(A.T) * 4);
    P.fg = make_rsrc(A.fpre + static_cast<int64_t>(s) * A.T, static_cast<uint32_t>(A.T) * 4);

    // ---- entry state ------------------------------------------------------------------------
    f32x16_t Cacc[8];
    const float* Cin = nullptr;
    const float* nin = nullptr;
    float m_prev;
    if (!FULL) {
        m_prev = -INFINITY;
    } else if (g == 0) {
        Cin = A.C0 ? A.C0 + static_cast<int64_t>(s) * kDQK * kDV : nullptr;
        nin = A.n0 ? A.n0 + static_cast<int64_t>(s) * kDQK : nullptr;
        m_prev = A.m0 ? A.m0[s] : 0.0f;
    } else {
        const float* slot = A.ws + (static_cast<int64_t>(s) * (A.G - 1) + (g - 1)) * kSlotFloats;
        Cin = slot;
        nin = slot + kDQK * kDV;
        m_prev = slot[kDQK * kDV + kDQK + 2];
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int d = 32 * dt + 8 * (j >> 2) + 4 * kg + (j & 3);
            Cacc[dt][j] = Cin ? Cin[static_cast<int64_t>(d) * kDV + v0 + 32 * wave + l32] : 0.0f;
        }
    }
    S.n[0][tid] = nin ? nin[tid] : 0.0f;
    if (tid == 0) S.scal[2] = 0.0f;

    VRegs<L> rv;
    QKRegs<L> rqk;
    if (c_begin < c_end) {
        load_v<L>(rv, P, c_begin * L, v0, tid);
        load_qk<L, FULL>(rqk, P, c_begin * L, 0, tid);
    }

    f32x16_t Nacc[NTT];
    f32x4_t Sacc[MAXT];
    float dq_part = 0.0f;

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * L;
        const int nb_cur = (c - c_begin) & 1;
        float* n_old = S.n[nb_cur];
        float* n_new = S.n[nb_cur ^ 1];
        __syncthreads();   // previous chunk fully consumed (Vt, St, gate vectors)
        if (wave == 0) gate_phase<L>(S, rv, m_prev, lane);
        store_v<L>(S, rv, tid);
        if (c + 1 < c_end) load_v<L>(rv, P, t0 + L, v0, tid);
        __syncthreads();
        const float decay = S.scal[0];
        const float m_next = S.scal[1];

        if constexpr (FULL) {
#pragma unroll
            for (int T = 0; T < NTT; ++T) Nacc[T] = f32x16_t{};
#pragma unroll
            for (int i = 0; i < MAXT; ++i) Sacc[i] = f32x4_t{};
            dq_part = 0.0f;
        }

#pragma unroll
        for (int p = 0; p < kNDB; ++p) {
            store_qk<L, FULL>(S, rqk, tid);
            __syncthreads();
            if (p + 1 < kNDB) {
                load_qk<L, FULL>(rqk, P, t0, p + 1, tid);
            } else if (c + 1 < c_end) {
                load_qk<L, FULL>(rqk, P, t0 + L, 0, tid);
            }

            if constexpr (FULL) {
                // (i) S^T += K_p Q_p^T on this wave's causal tiles
#pragma unroll
                for (int i = 0; i < MAXT; ++i) {
                    const int t = wave + kWaves * i;
                    if (t < NT_S) {
                        int tb = 0, rem = t;
                        while (rem > tb) { rem -= tb + 1; ++tb; }
                        const int sb = rem;
#pragma unroll
                        for (int ks = 0; ks < kDB / 32; ++ks) {
                            const u32x4_t a = *reinterpret_cast<const u32x4_t*>(&S.Kb[(16 * sb + l16) * QP + 32 * ks + 8 * g16]);
                            const u32x4_t b = *reinterpret_cast<const u32x4_t*>(&S.Qb[(16 * tb + l16) * QP + 32 * ks + 8 * g16]);
                            Sacc[i] = mfma16(a, b, Sacc[i]);
                        }
                    }
                }
                // (iii) N^T += C_p^T Q_p^T, A operand straight from the C accumulators
#pragma unroll
                for (int st = 0; st < 4; ++st) {
                    const f32x16_t& cc = Cacc[2 * p + (st >> 1)];
                    const int hh = st & 1;
                    u32x4_t a;
                    a[0] = pack_bf16x2(cc[8 * hh + 0], cc[8 * hh + 1]);
                    a[1] = pack_bf16x2(cc[8 * hh + 2], cc[8 * hh + 3]);
                    a[2] = pack_bf16x2(cc[8 * hh + 4], cc[8 * hh + 5]);
                    a[3] = pack_bf16x2(cc[8 * hh + 6], cc[8 * hh + 7]);
                    const int dl = 32 * (st >> 1) + 16 * hh + 4 * kg;
#pragma unroll
                    for (int T = 0; T < NTT; ++T) {
                        const uint16_t* qrow = &S.Qb[(32 * T + l32) * QP + dl];
                        u32x4_t b;
                        const u32x2_t b0 = *reinterpret_cast<const u32x2_t*>(qrow);
                        const u32x2_t b1 = *reinterpret_cast<const u32x2_t*>(qrow + 8);
                        b[0] = b0[0]; b[1] = b0[1]; b[2] = b1[0]; b[3] = b1[1];
                        Nacc[T] = mfma32(a, b, Nacc[T]);
                    }
                }
                // Q n_{k-1} partial over this d block (fp32 VALU)
                {
                    constexpr int TPR = kThreads / L;           // threads per row: 4 (L=64) or 2 (L=128)
                    constexpr int DPT = kDB / TPR;               // d per thread: 16 or 32
                    const int tau = tid / TPR, part = tid % TPR;
                    const uint16_t* qrow = &S.Qb[tau * QP + part * DPT];
                    const float* nrow = &n_old[p * kDB + part * DPT];
#pragma unroll
                    for (int e = 0; e < DPT; e += 8) {
                        const u32x4_t qq = *reinterpret_cast<const u32x4_t*>(qrow + e);
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            dq_part += lo_f32(qq[u]) * nrow[e + 2 * u] + hi_f32(qq[u]) * nrow[e + 2 * u + 1];
                    }
                }
            }

            // (iv) C_p = decay C_p + (w K)_p^T V
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) Cacc[2 * p + dt] *= decay;
#pragma unroll
            for (int ks = 0; ks < L / 16; ++ks) {
                const u32x4_t b = *reinterpret_cast<const u32x4_t*>(&S.Vt[(32 * wave + l32) * TP + 16 * ks + 8 * kg]);
#pragma unroll
                for (int dt = 0; dt < 2; ++dt) {
                    const u32x4_t a = *reinterpret_cast<const u32x4_t*>(&S.Ktb[(32 * dt + l32) * TP + 16 * ks + 8 * kg]);
                    Cacc[2 * p + dt] = mfma32(a, b, Cacc[2 * p + dt]);
                }
            }
            // n_p = decay n_p + K_p^T w  (fp32: exact bf16 K times fp32 w)
            {
                const int tp = tid & 7, dp = tid >> 3;   // 8 tau parts x 32 d pairs
                float s0 = 0.f, s1 = 0.f;
#pragma unroll
                for (int e = 0; e < L / 8; ++e) {
                    const int tau = tp * (L / 8) + e;
                    const uint32_t kk = *reinterpret_cast<const uint32_t*>(&S.Kb[tau * QP + 2 * dp]);
                    const float wt = S.w[tau];
                    s0 += wt * lo_f32(kk);
                    s1 += wt * hi_f32(kk);
                }
#pragma unroll
                for (int o = 1; o < 8; o <<= 1) {
                    s0 += __shfl_xor(s0, o, 64);
                    s1 += __shfl_xor(s1, o, 64);
                }
                if (tp == 0) {
                    const int d = p * kDB + 2 * dp;
                    n_new[d] = decay * n_old[d] + s0;
                    n_new[d + 1] = decay * n_old[d + 1] + s1;
                }
            }
            __syncthreads();
        }

        if constexpr (FULL) {
            // finish Q n
            {
                constexpr int TPR = kThreads / L;
#pragma unroll
                for (int o = 1; o < TPR; o <<= 1) dq_part += __shfl_xor(dq_part, o, 64);
                if ((tid % TPR) == 0) S.dq[tid / TPR] = dq_part;
            }
            // gate matrix on the S^T tiles -> S~ (bf16, tau-major) and row sums
#pragma unroll
            for (int i = 0; i < MAXT; ++i) {
                const int t = wave + kWaves * i;
                if (t < NT_S) {
                    int tb = 0, rem = t;
                    while (rem > tb) { rem -= tb + 1; ++tb; }
                    const int sb = rem;
                    const int tau = 16 * tb + l16;
                    const float Mt = S.M2[tau];
                    float vals[4];
                    float rsum = 0.f;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int sig = 16 * sb + 4 * g16 + j;
                        float val = 0.f;
                        if (sig <= tau) val = Sacc[i][j] * kQScale * fast_exp2(S.x2[sig] - Mt);
                        vals[j] = val;
                        rsum += val;
                    }
                    u32x2_t o;
                    o[0] = pack_bf16x2(vals[0], vals[1]);
                    o[1] = pack_bf16x2(vals[2], vals[3]);
                    *reinterpret_cast<u32x2_t*>(&S.St[tau * TP + 16 * sb + 4 * g16]) = o;
                    rsum += __shfl_xor(rsum, 16, 64);
                    rsum += __shfl_xor(rsum, 32, 64);
                    if (g16 == 0) S.rs[sb][tau] = rsum;
                }
            }
            // zero the masked 16x16 tiles inside each diagonal 32x32 block
            for (int T = wave; T < NTT; T += kWaves) {
                const int tau = 32 * T + l16;
                *reinterpret_cast<u32x2_t*>(&S.St[tau * TP + 32 * T + 16 + 4 * g16]) = u32x2_t{0u, 0u};
            }
            __syncthreads();
            // denominators
            if (tid < L) {
                const int tau = tid;
                float den = S.inter[tau] * S.dq[tau];
                for (int sb = 0; sb <= tau / 16; ++sb) den += S.rs[sb][tau];
                S.hinv[tau] = 1.0f / fmaxf(fabsf(den), S.floorv[tau]);
            }
            __syncthreads();
            // (ii) N^T = inter * N^T + V^T S~^T, then h
#pragma unroll
            for (int T = 0; T < NTT; ++T) {
                const int tau = 32 * T + l32;
                Nacc[T] *= S.inter[tau];
#pragma unroll
                for (int ks = 0; ks < 2 * T + 2; ++ks) {
                    const u32x4_t a = *reinterpret_cast<const u32x4_t*>(&S.Vt[(32 * wave + l32) * TP + 16 * ks + 8 * kg]);
                    const u32x4_t b = *reinterpret_cast<const u32x4_t*>(&S.St[tau * TP + 16 * ks + 8 * kg]);
                    Nacc[T] = mfma32(a, b, Nacc[T]);
                }
                const float hv = S.hinv[tau];
                uint16_t* hrow = A.h + (static_cast<int64_t>(s) * A.T + t0 + tau) * kDV + v0 + 32 * wave + 4 * kg;
#pragma unroll
                for (int jg = 0; jg < 4; ++jg) {
                    u32x2_t o;
                    o[0] = pack_bf16x2(Nacc[T][4 * jg + 0] * hv, Nacc[T][4 * jg + 1] * hv);
                    o[1] = pack_bf16x2(Nacc[T][4 * jg + 2] * hv, Nacc[T][4 * jg + 3] * hv);
                    *reinterpret_cast<u32x2_t*>(hrow + 8 * jg) = o;
                }
            }
        }
        m_prev = m_next;
    }
    __syncthreads();

    // ---- exit state ---------------------------------------------------------------------------
    const int nfinal = (c_end - c_begin) & 1;
    float* Cout;
    float* nout;
    float* mout;
    bool write_nm = (tile == 0);
    if (FULL) {
        if (g != A.G - 1) return;
        Cout = A.CT + static_cast<int64_t>(s) * kDQK * kDV;
        nout = A.nT + static_cast<int64_t>(s) * kDQK;
        mout = A.mT + s;
    } else {
        float* slot = A.ws + (static_cast<int64_t>(s) * (A.G - 1) + g) * kSlotFloats;
        Cout = slot;
        nout = slot + kDQK * kDV;
        mout = nout + kDQK;   // m_loc, then gsum
        if (write_nm && tid == 0) mout[1] = S.scal[2];
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int d = 32 * dt + 8 * (j >> 2) + 4 * kg + (j & 3);
            Cout[static_cast<int64_t>(d) * kDV + v0 + 32 * wave + l32] = Cacc[dt][j];
        }
    }
    if (write_nm) {
        nout[tid] = S.n[nfinal][tid];
        if (tid == 0) mout[0] = m_prev;
    }
}

// Entry states of segments 1..G-1 from the local segment states (in place).
__global__ void __launch_bounds__(256) combine_kernel(float* ws, const float* C0, const float* n0, const float* m0,
                                                      int G) {
    const int s = blockIdx.y;
    float* base = ws + static_cast<int64_t>(s) * (G - 1) * kSlotFloats;
    // scalar chain of entry max states (every block computes it; block 0 stores it)
    float m_in = m0 ? m0[s] : 0.0f;
    constexpr int kE4 = (kDQK * kDV + kDQK) / 4;
    const int e4 = blockIdx.x * blockDim.x + threadIdx.x;
    float4 cur = make_float4(0.f, 0.f, 0.f, 0.f);
    if (e4 < kE4) {
        if (e4 < kDQK * kDV / 4) {
            if (C0) cur = reinterpret_cast<const float4*>(C0 + static_cast<int64_t>(s) * kDQK * kDV)[e4];
        } else if (n0) {
            cur = reinterpret_cast<const float4*>(n0 + static_cast<int64_t>(s) * kDQK)[e4 - kDQK * kDV / 4];
        }
    }
    for (int gg = 0; gg < G - 1; ++gg) {
        float* slot = base + static_cast<int64_t>(gg) * kSlotFloats;
        const float m_loc = slot[kDQK * kDV + kDQK];
        const float gsum = slot[kDQK * kDV + kDQK + 1];
        const float m_new = fmaxf(gsum + m_in, m_loc);
        const float a = expf(gsum + m_in - m_new);
        const float b = expf(m_loc - m_new);
        if (e4 < kE4) {
            float4* p4 = reinterpret_cast<float4*>(slot) + e4;
            const float4 loc = *p4;
            cur.x = a * cur.x + b * loc.x;
            cur.y = a * cur.y + b * loc.y;
            cur.z = a * cur.z + b * loc.z;
            cur.w = a * cur.w + b * loc.w;
            *p4 = cur;
        }
        if (blockIdx.x == 0 && threadIdx.x == 0) slot[kDQK * kDV + kDQK + 2] = m_new;
        m_in = m_new;
    }
}

template <int L>
size_t smem_bytes() {
    return sizeof(Smem<L>);
}

template <int L, bool FULL>
hipError_t launch_variant(const ChunkKernelArgs& a, int S, hipStream_t stream) {
    const size_t lds = smem_bytes<L>();
    auto kern = chunk_mfma_kernel<L, FULL>;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int G_run = FULL ? a.G : a.G - 1;
    const dim3 grid(static_cast<unsigned>(S * G_run * kNTile));
    hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, stream, a);
    return hipGetLastError();
}

}  // namespace

bool chunk_mfma_supported(mlstm_dtype dt, int DQK, int DV, int L) {
    return dt == MLSTM_BF16 && DQK == kDQK && DV == kDV && (L == 64 || L == 128);
}

int chunk_mfma_segments(int B, int NH, int T, int L) {
    const int S = B * NH;
    const int nc = T / L;
    if (nc <= 1) return 1;
    const int wgs = S * kNTile;
    constexpr int kTargetWGs = 256;
    int G = (kTargetWGs + wgs - 1) / wgs;
    if (G > nc / 2) G = nc / 2;   // at least two chunks per segment
    if (G < 1) G = 1;
    const int seg = (nc + G - 1) / G;
    return (nc + seg - 1) / seg;
}

size_t chunk_mfma_workspace_bytes(int B, int NH, int T, int DQK, int DV, int L) {
    (void)DQK;
    (void)DV;
    const int G = chunk_mfma_segments(B, NH, T, L);
    if (G <= 1) return 0;
    return static_cast<size_t>(B) * NH * (G - 1) * kSlotFloats * sizeof(float);
}

hipError_t launch_chunk_mfma(const ChunkArgs& a, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    const int S = a.B * a.NH;
    const int nc = a.T / a.L;
    int G = workspace ? chunk_mfma_segments(a.B, a.NH, a.T, a.L) : 1;
    if (G > 1 && workspace_bytes < chunk_mfma_workspace_bytes(a.B, a.NH, a.T, a.DQK, a.DV, a.L)) G = 1;
    if (nc == 0) G = 1;
    const int seg_chunks = G > 1 ? (nc + G - 1) / G : nc;

    ChunkKernelArgs k{};
    k.q = static_cast<const uint16_t*>(a.q);
    k.k = static_cast<const uint16_t*>(a.k);
    k.v = static_cast<const uint16_t*>(a.v);
    k.ipre = a.ipre;
    k.fpre = a.fpre;
    k.C0 = a.C0;
    k.n0 = a.n0;
    k.m0 = a.m0;
    k.ws = static_cast<float*>(workspace);
    k.T = a.T;
    k.G = G;
    k.seg_chunks = seg_chunks;
    k.h = static_cast<uint16_t*>(a.h);
    k.CT = a.CT;
    k.nT = a.nT;
    k.mT = a.mT;

    hipError_t e;
    if (G > 1) {
        e = (a.L == 64) ? launch_variant<64, false>(k, S, stream) : launch_variant<128, false>(k, S, stream);
        if (e != hipSuccess) return e;
        constexpr int kE4 = (kDQK * kDV + kDQK) / 4;
        hipLaunchKernelGGL(combine_kernel, dim3((kE4 + 255) / 256, S), dim3(256), 0, stream, k.ws, a.C0, a.n0, a.m0,
                           G);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return (a.L == 64) ? launch_variant<64, true>(k, S, stream) : launch_variant<128, true>(k, S, stream);
}

}  // namespace mlstm
