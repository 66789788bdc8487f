// Device pieces shared by the chunkwise prefill kernel and the backward's chunk walk (bf16, the
// xLSTM 7B head shape): the workgroup shape, the chunk configuration, the per-chunk gate quantities
// and the gate phase that computes them, V staging with its transposition on the matrix cores, and
// the sequence addressing.  Everything lives in an anonymous namespace, so each translation unit that
// includes this header has its own copy.
#pragma once
#include "mfma_common.h"

namespace mlstm {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = 8;
constexpr int kGateWave = kWaves - 1; // the wave with the least MFMA work runs the gate scans
constexpr float kRenorm = -20.0f;     // rescale C eagerly when its lazy log-scale would drop below this

template <int L>
struct Cfg {
    static constexpr int NDB = (L == 128) ? 4 : 2;  // d blocks staged per chunk
    static constexpr int DB = kDQK / NDB;           // 128 or 64
    static constexpr int DT = DB / 16;              // 16-row C tiles per d block
    // row pitch (elements) of Q and K blocks: 288 bytes (L = 64) or 160 bytes (L = 128) keep the
    // 16-byte row reads of 16 consecutive rows free of bank conflicts (a 144-byte pitch measured 1.6%
    // slower on the B = 4 x T = 32768 prefill)
    static constexpr int QP = DB + 16;
    static constexpr int SP = (L == 64) ? L + 16 : L + 8;   // row pitch of S~ (160 bytes at L = 64)
    static constexpr int NB = L / 16;               // 16-wide blocks along the chunk
    static constexpr int QKE = L * QP;              // elements of one Q or K block buffer
    // L = 128: S~ lives in the second Q/K buffer set, which is free from the end of the
    // chunk's last d block to the next chunk's first store into it; this keeps the
    // workgroup within the 160 KB of LDS
    static constexpr bool ST_ALIAS = (L == 128);
    // Wave split of the workgroup's 256 x 128 slice of C: DH d partitions x (8 / DH) column
    // groups of VT = DH 16-column tiles.  DH = 2 (L = 64) halves the Q and K^T operand reads of
    // (iii) and (iv) at the price of summing the two partial read-outs of (iii) through LDS;
    // L = 128 keeps DH = 1 (its read-out accumulators would not fit twice).
    static constexpr int DH = (L == 64) ? 2 : 1;
    static constexpr int VT = DH;
    static constexpr int NVG = kWaves / DH;
    // V is kept in LDS transposed (rows v, tau contiguous, pitch TP), once plain for (ii) and once
    // scaled by the C-update key weights for (iv), so both read it with plain 16-byte row reads
    static constexpr int TP = L + 8;
    // L = 128 stages K only transposed (K^T rows [d][tau], pitch KTP, transposed on the matrix cores
    // like V): (iv) and the n update read it with 16-byte row reads, (i) with transpose reads.  L = 64
    // stages K rows (its LDS holds no room for a second layout next to the read-out exchange).
    static constexpr bool KT = (L == 128);
    static constexpr int KTP = L + 8;
    static constexpr int KTE = DB * KTP;
    static constexpr int SETE = QKE + (KT ? KTE : QKE);   // elements of one d-block set: Q, then K
};

// Physical K^T row of d (within a d block): bit 2 flipped when bit 4 is set, so that the 16 rows an
// (iv) operand reads (d = 32 pp + 8 i + 4 e + 0..3, i = 0..3) and the 16 consecutive rows an n-update
// operand reads fall in 16 different 4-bank groups at a 272-byte pitch; four consecutive d stay
// consecutive (the transpose reads of (i) take them four at a time).
__device__ __forceinline__ int kt_row(int d) { return d ^ (((d >> 4) & 1) << 2); }

// Per-chunk gate quantities, written one chunk ahead by the gate wave.
template <int L>
struct alignas(16) GateBuf {
    float x2[L];        // (i~ - b) * log2 e
    float M2[L];        // M * log2 e (0 for a row with no input at all)
    int R[L];           // last restart (forget gate exactly zero) at or before the row, -1: none
    float interC[L];    // exp(m_prev - M + s) / sqrt(DQK): scale of C_acc^T Q^T
    float interN[L];    // exp(m_prev - M) / sqrt(DQK):     scale of Q n
    float floorv[L];    // exp(-(b + M))
    float wC[L];        // C-update weights exp(x - M_L - s_new)
    uint16_t wb[2][L];  // n-update weights exp(x - M_L) as bf16 hi / lo rows
    float scal[4];      // [0] n decay, [1] m_next, [2] s_new, [3] eager C scale (1: none)
};

// V is staged in VPARTS parts (two at L = 128, whose four d blocks leave time for it) so
// that fewer registers hold it at once.
template <int L>
struct VRegs {
    static constexpr int PARTS = (Cfg<L>::NDB >= 3) ? 2 : 1;
    static constexpr int N = (L * kDVT / 8) / kThreads / PARTS;   // pieces per thread per part
    u32x4_t v[N];
};

// V pieces in the MFMA A-operand layout for vt_transpose: for piece i of part `part`, lane (l16, g16)
// of wave w holds V[tau 16 a + l16][v 32 b + 8 g16 + 0..7] with pc = w + 8 (part N + i) and
// (a, b) = (pc % (L / 16), pc / (L / 16)), so the workgroup's pieces cover the L x 128 chunk once.
template <int L>
__device__ __forceinline__ void load_v_tr(VRegs<L>& r, const SeqRsrc& R, int t0, int v0, int wave, int lane, int part,
                                          uint32_t rv) {
    constexpr int NW = kWaves;
    static_assert(VRegs<L>::PARTS * VRegs<L>::N * NW == (L / 16) * (kDVT / 32), "pieces of one L x 128 chunk");
    constexpr int NA = L / 16;
    const uint32_t soff = v0 * 2;   // the row offset goes in the per-lane offset
    int ln = lane;   // opaque: the offsets are recomputed per call rather than held across the loop
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int i = 0; i < VRegs<L>::N; ++i) {
        const int pc = wave + NW * (part * VRegs<L>::N + i), a = pc % NA, b = pc / NA;
        r.v[i] = bload128(R.v, static_cast<uint32_t>(t0 + 16 * a + (ln & 15)) * rv + (32 * b + 8 * (ln >> 4)) * 2, soff);
    }
}
template <int L>
using VtPacked = u32x2_t[2 * VRegs<L>::N * VRegs<L>::PARTS];
// The transposition on the matrix cores: D = A E_h with A a piece (16 tau x 32 v) and E_h the 32 x 16
// one-hot selection of its columns 16 h + 0..15 (exact in fp32).  Lane (n = l16, g16) of D holds
// V[tau 16 a + 4 g16 + j][v 32 b + 16 h + n], j = 0..3: four consecutive tau of one row of V^T, kept
// packed in pv until the stores below.
// One-hot selection E_h (32 x 16, columns 16 h + 0..15 of a 32-column piece) in the B-operand layout:
// lane (l16, g16) holds k slots 8 g16 + 0..7 of column l16, whose one (if any) is slot 16 h + l16.
// That slot lies in the lane's eight when 16 h + l16 - 8 g16 is in 0..7, i.e. when g16 = 2 h + l16 / 8,
// and is then slot l16 % 8 of them: register (l16 / 2) % 4, half l16 % 2.  Built from an opaque copy
// of the lane index so that it is not hoisted out of the chunk loop (eight more registers held
// across the loop would spill).
__device__ __forceinline__ void onehot_pair(u32x4_t (&E)[2], int lane) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int sel = (ln >> 1) & 3;
    const int gh = (ln >> 4) - ((ln >> 3) & 1);   // 2 h for the h whose column this lane can hold
    const uint32_t one = (ln & 1) ? 0x3F800000u : 0x3F80u;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t oh = (gh == 2 * h) ? one : 0u;
#pragma unroll
        for (int d = 0; d < 4; ++d) E[h][d] = (sel == d) ? oh : 0u;
    }
}

template <int L>
__device__ __forceinline__ void vt_transpose(VtPacked<L>& pv, const VRegs<L>& r, int lane, int part) {
    u32x4_t E[2];
    onehot_pair(E, lane);
#pragma unroll
    for (int i = 0; i < VRegs<L>::N; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const f32x4_t d = mfma16(r.v[i], E[h], f32x4_t{});
            pv[2 * (part * VRegs<L>::N + i) + h] = u32x2_t{pack_bf16x2(d[0], d[1]), pack_bf16x2(d[2], d[3])};
        }
}

template <int L>
__device__ __forceinline__ void load_gates(float (&gi)[2], float (&gf)[2], const SeqRsrc& R, int t0, int lane) {
    const uint32_t goff = static_cast<uint32_t>(t0 + lane) * 4;   // range-checked: zero past the end
    gi[0] = bloadf(R.ig, goff, 0);
    gf[0] = bloadf(R.fg, goff, 0);
    if constexpr (L == 128) {
        gi[1] = bloadf(R.ig, goff + 256, 0);
        gf[1] = bloadf(R.fg, goff + 256, 0);
    }
}


// Gate phase of one chunk (run by one wave): in-chunk prefix sums and maxima, the max
// state, the lazy C scale, and every per-row scale of the chunk.  m_prev and s_cur
// carry the max state and the lazy log-scale from chunk to chunk.  Rows at or beyond
// nvalid (the partial last chunk of a sequence) are neutral tokens: no input (x = -inf)
// and no decay (logsig f~ = 0), so they leave the state unchanged.
//
// A forget gate of exactly zero (f~ = -inf, a document border) restarts the state: nothing
// before that token reaches it or any later token.  The prefix sum b skips the restart token
// (the decay from s to t over tokens s+1..t never includes a restart for the pairs that
// survive), every row keeps R, its last restart at or before it, and the row's maxima, weights
// and entry-state terms cover only the tokens from R on.  A chunk that holds a restart drops
// its entry state: C and n are scaled by zero before this chunk's keys are added.
template <int L>
__device__ __forceinline__ void gate_phase(GateBuf<L>& Gb, const float (&gi)[2], const float (&gf)[2], float& m_prev,
                                           float& s_cur, int lane, int nvalid) {
    const bool ok0 = lane < nvalid;
    const float lg0 = ok0 ? flogsig(gf[0]) : 0.0f;
    const bool rs0 = (lg0 == -INFINITY);
    bool rs1 = false;
    float lg1 = 0.f;
    if constexpr (L == 128) {
        lg1 = (64 + lane < nvalid) ? flogsig(gf[1]) : 0.0f;
        rs1 = (lg1 == -INFINITY);
    }
    // restarts are rare: a chunk without one (a wave-uniform test) takes the plain scans
    const bool any_restart = __builtin_amdgcn_ballot_w64(rs0 || rs1) != 0;
    const float b = wave_incl_sum(rs0 ? 0.0f : lg0);
    const float x = ok0 ? gi[0] - b : -INFINITY;
    float r = -1.f, p;
    if (any_restart) {
        r = wave_incl_max(rs0 ? static_cast<float>(lane) : -1.0f);
        p = wave_seg_incl_max(x, rs0);
    } else {
        p = wave_incl_max(x);
    }
    float b2 = 0.f, x2 = 0.f, p2 = 0.f, r2 = -1.f;
    if constexpr (L == 128) {
        const bool ok1 = 64 + lane < nvalid;
        b2 = lane63(b) + wave_incl_sum(rs1 ? 0.0f : lg1);
        x2 = ok1 ? gi[1] - b2 : -INFINITY;
        if (any_restart) {
            const float r_own = wave_incl_max(rs1 ? static_cast<float>(64 + lane) : -1.0f);
            r2 = fmaxf(lane63(r), r_own);
            const float q2 = wave_seg_incl_max(x2, rs1);
            p2 = (r_own >= 0.0f) ? q2 : fmaxf(lane63(p), q2);
        } else {
            p2 = fmaxf(lane63(p), wave_incl_max(x2));
        }
    }
    const float pL = lane63(L == 128 ? p2 : p);
    const float bL = lane63(L == 128 ? b2 : b);
    const float rL = lane63(L == 128 ? r2 : r);
    const bool restart = (rL >= 0.0f);
    const float ML = restart ? pL : fmaxf(m_prev, pL);
    // an empty state (m = -inf) has nothing to decay, and a restart drops the state
    const bool empty = restart || (m_prev == -INFINITY);
    const float dlog = empty ? 0.0f : m_prev - ML;
    const float s_try = s_cur + dlog;
    const bool eager = restart || s_try < kRenorm;
    const float s_new = eager ? 0.0f : s_try;
    auto emit = [&](int tau, float bb, float xx, float pp, float rr) {
        const bool fresh = (rr >= 0.0f);   // a restart at or before this row: no entry-state term
        const float M = fresh ? pp : fmaxf(m_prev, pp);
        Gb.x2[tau] = xx * kLog2e;
        Gb.M2[tau] = (M == -INFINITY) ? 0.0f : M * kLog2e;
        Gb.R[tau] = static_cast<int>(rr);
        Gb.interC[tau] = (fresh || M == -INFINITY) ? 0.0f : fexp(m_prev - M + s_cur) * kQScale;
        Gb.interN[tau] = (fresh || M == -INFINITY) ? 0.0f : fexp(m_prev - M) * kQScale;
        Gb.floorv[tau] = fexp(-(bb + M));
        const bool none = (xx == -INFINITY) || (static_cast<float>(tau) < rL);
        Gb.wC[tau] = none ? 0.0f : fexp(xx - ML - s_new);
        const float wn = none ? 0.0f : fexp(xx - ML);
        const uint16_t whi = f32_to_bf16(wn);
        Gb.wb[0][tau] = whi;
        Gb.wb[1][tau] = f32_to_bf16(wn - bf16_to_f32(whi));
    };
    emit(lane, b, x, p, r);
    if constexpr (L == 128) emit(64 + lane, b2, x2, p2, r2);
    const float m_next = bL + ML;
    if (lane == 0) {
        Gb.scal[0] = (empty || ML == -INFINITY) ? 0.0f : fexp(m_prev - ML);
        Gb.scal[1] = m_next;
        Gb.scal[2] = s_new;
        Gb.scal[3] = restart ? 0.0f : (eager ? fexp(s_try) : 1.0f);
    }
    m_prev = m_next;
    s_cur = s_new;
}

// First row of sequence s = (batch b, head s - b NH), written as s st_h + b (st_b - NH st_h) with
// st = {st_b - NH st_h, st_h}, and the byte span of its T rows of D elements.  b = floor(s / NH)
// comes from a multiply by the host's nh_magic (nh_magic = 0 stands for NH = 1, b = s): it is exact
// while s NH < 2^32 (the host checks this for strided calls), and contiguous rows have st[0] = 0.
// (An integer division, the form b st_b + (s - b NH) st_h, and this helper itself in the chunk
// kernel all made the compiler's code for its chunk loop markedly slower; the chunk kernel writes the
// same sum out in place.)
__device__ __forceinline__ const uint16_t* seq_rows(const uint16_t* p, int s, uint32_t nh_magic, const int64_t (&st)[2]) {
    const int b = nh_magic ? static_cast<int>(__umulhi(static_cast<uint32_t>(s), nh_magic)) : s;
    return p + static_cast<int64_t>(s) * st[1] + static_cast<int64_t>(b) * st[0];
}
__device__ __forceinline__ uint32_t seq_span(int T, uint32_t row_bytes, int D) {
    return T > 0 ? static_cast<uint32_t>(T - 1) * row_bytes + static_cast<uint32_t>(D) * 2u : 0u;
}

}  // namespace
}  // namespace mlstm
