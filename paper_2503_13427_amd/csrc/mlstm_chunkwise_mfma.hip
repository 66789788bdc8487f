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
// Lazily scaled matrix memory.  The accumulators hold C_acc with C = C_acc e^{s}.
// A chunk's decay is folded into s (s += m_prev - M_L) and into the key weights
// of the update (w e^{-s} <= e^{-kRenorm}), so the 64 accumulator registers of C in
// a wave are not rescaled by VALU work in most chunks; when s would fall below
// kRenorm the chunk applies the decay eagerly instead (C_acc *= e^{s + m_prev - M_L},
// between the read-out (iii) and the update (iv)) and s returns to 0.  The
// inter-chunk term uses exp(m_prev - M_tau + s); the exit state is C_acc e^{s}.
//
// Products and their MFMA mapping (gfx950 bf16 16x16x32 MFMA, fp32 accumulate):
//   (i)   S^T = K Q^T             A = K rows, B = Q rows (both d-contiguous)
//   (ii)  N^T += V^T S~^T         A = V^T rows, B = S~ rows
//   (iii) N^T += C^T Q^T          A = the C accumulators of (iv), converted to bf16 in
//                                 registers, B = Q rows
//   (iv)  C += K^T (w e^{-s} V)   A = K read transposed, B = (w e^{-s} V)^T rows
//   Q n and K^T w                 the fp32 normaliser and weights split into bf16 hi + lo
//                                 rows (relative error ~2^-17)
// "Read transposed" is the LDS transpose read of gfx950 (ds_read_b64_tr_b16): in each
// 16-lane group, lane 4s+q supplies 4 consecutive elements of row s of a 4 x 16 tile and
// lane c receives column c, so a row-major [k][m] tile arrives k-contiguous, as an MFMA
// operand wants it.  Q and K live in LDS in their natural layout.  V is transposed once per
// chunk on the matrix cores instead (a piece in the A-operand layout times a one-hot
// selection, exact) and kept in LDS as V^T and as the key-weighted (w e^{-s} V)^T, so (ii)
// and (iv) read it with plain 16-byte row reads.
// (iii) consumes C in the accumulator layout of (iv): the contraction index d is
// permuted consistently in both operands.  Outputs come out transposed (rows v,
// columns tau), so each lane stores runs of four consecutive v of one h row.
//
// Work decomposition.  One workgroup of 8 waves (two per SIMD, so one wave's
// LDS and memory waits are covered by the other's MFMAs) owns one (sequence,
// 128-column dv tile, segment) and walks the segment's chunks in order.  Each wave
// owns 64 accumulator registers of C for the whole segment (L = 64: a 128 x 32 slice,
// one of two d partitions of a 32-column group; L = 128: a 256 x 16 slice); S~, Q n
// and the gates are computed once per workgroup.
// Q and K are staged in d blocks (two of 128 for L = 64, four of 64 for L = 128);
// the next block (and the next chunk's V and gates) is prefetched into registers
// while the current block is multiplied.  The four dv tiles of a (sequence,
// segment) are dispatched consecutively onto one XCD so their shared Q/K reads
// hit one L2.
//
// Segment-parallel schedule (optional workspace).  With G segments per sequence:
// (1) local_state_kernel computes the state of each of the first G-1 segments (split
// into R sub-segments of at most kLocMax tokens) from an empty state, as one weighted
// contraction over its tokens; (2) a combine kernel scans those local states into each
// segment's entry state, m_in' = max(gsum + m_in, m_loc),
// C_in' = e^{gsum + m_in - m_in'} C_in + e^{m_loc - m_in'} C_loc; (3) the chunkwise
// kernel runs every segment from its entry state.
#include <mutex>

#include "chunk_common.h"
#include "launch.h"

namespace mlstm {
namespace {

template <int L>
struct Smem {
    using C = Cfg<L>;
    // d-block set s: Q [tau * QP + d], then K (L = 64: rows [tau * QP + d]; L = 128: K^T
    // [kt_row(d) * KTP + tau]); d block p uses set p % 2
    uint16_t QK[2][C::SETE];
    // [0] V^T[v][tau] and [1] (w e^{-s} V)^T[v][tau] of the current chunk (this workgroup's 128 columns)
    uint16_t Vs[2][kDVT * C::TP];
    uint16_t St_own[C::ST_ALIAS ? 8 : L * C::SP];  // S~[tau][sig] when it has its own buffer
    uint16_t nb[2][2][kDQK];                       // normaliser as bf16 hi / lo rows, double-buffered
    float n[2][kDQK];                              // fp32 normaliser, double-buffered across chunks
    float dq[L];                                   // Q n_{k-1} (unscaled q)
    // row sums of S~ per (sigma block, tau): at L = 128 tau-major, so (ii) reads a row's eight in two
    // 16-byte reads; at L = 64 sigma-block-major (measured faster there)
    alignas(16) float rs[L * (L / 16)];
    __device__ float& rsum_at(int tau, int sb) { return rs[L == 128 ? tau * (L / 16) + sb : sb * L + tau]; }
    GateBuf<L> G[2];                               // by chunk parity
    // partial read-outs exchanged between the two d partitions of a column group (DH = 2):
    // [column group][v tile][tau tile][lane] as float4
    float X[C::DH == 2 ? C::NVG * C::VT * (L / 16) * 64 * 4 : 4];
};
static_assert(Cfg<128>::ST_ALIAS && 128 * Cfg<128>::SP <= Cfg<128>::SETE, "S~ must fit in one Q/K set");
static_assert(sizeof(Smem<64>) <= 160 * 1024 && sizeof(Smem<128>) <= 160 * 1024, "LDS budget");

// Per-thread staging registers: one Q/K d block in flight (V: VRegs).
template <int L>
struct QKRegs {
    static constexpr int N = (L * Cfg<L>::DB / 8) / kThreads;   // 16-byte pieces per thread per matrix
    u32x4_t q[N];
    u32x4_t k[N];
};


// Q and K rows are 512 bytes, V rows 1024 bytes; offsets are in bytes.
// With K^T staging (L = 128) K is loaded in pieces in the MFMA A-operand layout: piece i of wave w
// (pc = w + 8 i, a = pc % (L / 16), b = pc / (L / 16)) has lane (l16, g16) holding
// K[tau 16 a + l16][d 32 b + 8 g16 + 0..7] of the d block.
// The chunk's row offset t0 rides in the per-lane offset with the row, so rows past the end of a
// sequence fall outside the buffer range and read as zero in a partial last chunk; the scalar offset
// carries only the column base.  Row strides (bytes) come from the call: q, k and v may be strided
// views of one projection output.
template <int L>
__device__ __forceinline__ void load_qk(QKRegs<L>& r, const SeqRsrc& R, int t0, int p, int tid, uint32_t rq,
                                        uint32_t rk) {
    constexpr int NW = kWaves;
    constexpr int DB = Cfg<L>::DB, PR = DB / 8;   // 16-byte pieces per row
    const uint32_t soff = p * (DB * 2);
#pragma unroll
    for (int i = 0; i < QKRegs<L>::N; ++i) {
        const int item = tid + i * kThreads;
        const uint32_t row = static_cast<uint32_t>(t0 + item / PR), col = 16 * (item % PR);
        r.q[i] = bload128(R.q, row * rq + col, soff);
        if constexpr (!Cfg<L>::KT) r.k[i] = bload128(R.k, row * rk + col, soff);
    }
    if constexpr (Cfg<L>::KT) {
        static_assert(QKRegs<L>::N * NW == (L / 16) * (DB / 32), "pieces of one K block");
        int ln = tid & 63;   // opaque: recomputed per call rather than held across the loop
        asm volatile("" : "+v"(ln));
        const int wave = tid >> 6;
#pragma unroll
        for (int i = 0; i < QKRegs<L>::N; ++i) {
            const int pc = wave + NW * i, a = pc % (L / 16), b = pc / (L / 16);
            r.k[i] = bload128(R.k, static_cast<uint32_t>(t0 + 16 * a + (ln & 15)) * rk + (32 * b + 8 * (ln >> 4)) * 2,
                              soff);
        }
    }
}
template <int L>
__device__ __forceinline__ void store_qk(uint16_t* Qd, uint16_t* Kd, const QKRegs<L>& r, int tid) {
    constexpr int PR = Cfg<L>::DB / 8, QP = Cfg<L>::QP, NW = kWaves;
#pragma unroll
    for (int i = 0; i < QKRegs<L>::N; ++i) {
        const int item = tid + i * kThreads;
        const int off = (item / PR) * QP + 8 * (item % PR);
        MLSTM_CHECK(off >= 0 && off + 8 <= Cfg<L>::QKE, kDbgChunkMfma);
        *reinterpret_cast<u32x4_t*>(&Qd[off]) = r.q[i];
        if constexpr (!Cfg<L>::KT) *reinterpret_cast<u32x4_t*>(&Kd[off]) = r.k[i];
    }
    if constexpr (Cfg<L>::KT) {
        // K^T on the matrix cores: D = (piece) E_h holds, in lane (n = l16, g16), K[tau 16 a + 4 g16 + j]
        // [d 32 b + 16 h + n], j = 0..3 (exact), stored as four consecutive tau of K^T row d
        constexpr int KTP = Cfg<L>::KTP;
        const int lane = tid & 63, wave = tid >> 6;
        u32x4_t E[2];
        onehot_pair(E, lane);
        const int l16 = lane & 15, g16 = lane >> 4;
#pragma unroll
        for (int i = 0; i < QKRegs<L>::N; ++i) {
            const int pc = wave + NW * i, a = pc % (L / 16), b = pc / (L / 16);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const f32x4_t d = mfma16(r.k[i], E[h], f32x4_t{});
                const u32x2_t o{pack_bf16x2(d[0], d[1]), pack_bf16x2(d[2], d[3])};
                MLSTM_CHECK(kt_row(32 * b + 16 * h + l16) < Cfg<L>::DB && 16 * a + 4 * g16 + 4 <= KTP, kDbgChunkMfma);
                *reinterpret_cast<u32x2_t*>(&Kd[kt_row(32 * b + 16 * h + l16) * KTP + 16 * a + 4 * g16]) = o;
            }
        }
    }
}
// (w V)^T from the packed V^T: row weights wC of the chunk, rounded to bf16 once
template <int L>
__device__ __forceinline__ void vt_store_scaled(uint16_t* VwT, const VtPacked<L>& pv, const float* wC, int wave,
                                                int lane) {
    constexpr int TP = Cfg<L>::TP, NA = L / 16, NW = kWaves;
    const int l16 = lane & 15, g16 = lane >> 4;
#pragma unroll
    for (int i = 0; i < VRegs<L>::N * VRegs<L>::PARTS; ++i) {
        const int pc = wave + NW * i, a = pc % NA, b = pc / NA;
        const int tau = 16 * a + 4 * g16;
        const f32x4_t w = *reinterpret_cast<const f32x4_t*>(&wC[tau]);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const u32x2_t x = pv[2 * i + h];
            u32x2_t o;
            o[0] = pack_bf16x2(lo_f32(x[0]) * w[0], hi_f32(x[0]) * w[1]);
            o[1] = pack_bf16x2(lo_f32(x[1]) * w[2], hi_f32(x[1]) * w[3]);
            MLSTM_CHECK(32 * b + 16 * h + l16 < kDVT && tau + 4 <= TP, kDbgChunkMfma);
            *reinterpret_cast<u32x2_t*>(&VwT[(32 * b + 16 * h + l16) * TP + tau]) = o;
        }
    }
}
template <int L>
__device__ __forceinline__ void vt_store_plain(uint16_t* VtT, const VtPacked<L>& pv, int wave, int lane) {
    constexpr int TP = Cfg<L>::TP, NA = L / 16, NW = kWaves;
    const int l16 = lane & 15, g16 = lane >> 4;
#pragma unroll
    for (int i = 0; i < VRegs<L>::N * VRegs<L>::PARTS; ++i) {
        const int pc = wave + NW * i, a = pc % NA, b = pc / NA;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            MLSTM_CHECK(32 * b + 16 * h + l16 < kDVT && 16 * a + 4 * g16 + 4 <= TP, kDbgChunkMfma);
            *reinterpret_cast<u32x2_t*>(&VtT[(32 * b + 16 * h + l16) * TP + 16 * a + 4 * g16]) = pv[2 * i + h];
        }
    }
}
// Gate pre-activations of one chunk, one (L = 64) or two (L = 128) per lane of the gate wave.


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
    int S;             // sequences (B NH)
    int T;
    int G;             // segments per sequence
    int R;             // local sub-segments per segment; segment g >= 1 enters from slot g R - 1
    int NS;            // local slots per sequence, (G - 1) R
    int seg_chunks;    // chunks per segment (last may be shorter)
    uint16_t* h;
    float* CT;
    float* nT;
    float* mT;
    uint32_t nh_magic;             // floor(2^32 / NH) + 1, or 0 for NH = 1 (see seq_rows)
    // element strides of q, k, v: [0] batch stride - NH head stride, [1] head stride (see seq_rows)
    int64_t sq[2], sk[2], sv[2];
    uint32_t rq, rk, rv;           // their row (token) strides in bytes
};


// row pitch (floats) of the entry-state staging of a 256 x 128 tile in LDS: 528 bytes puts the
// rows 8 apart that one read of the accumulator pickup touches in different banks
constexpr int kStageP = kDVT + 4;
static_assert(kDQK * kStageP * 4 <= sizeof(Smem<64>) && kDQK * kStageP * 4 <= sizeof(Smem<128>), "staging");


// Staging order (one Q/K block and one part of a V chunk in registers at a time): block 0
// of a chunk is stored during the previous chunk (at the barrier that opens its last d
// block), block 1 at the top of the chunk, block p + 1 (p >= 1) at the barrier that opens
// block p.  The next chunk's V is loaded from the top of a chunk on, part k transposed in
// registers at the barrier that opens d block k + 1; its weighted copy goes to LDS after the
// S~ barrier (once this chunk's (iv) is done and the next chunk's weights are known), its
// plain copy at the top of the next chunk (once this chunk's (ii) is done).
template <int L>
__global__ void __launch_bounds__(kThreads, 1) chunk_mfma_kernel(ChunkKernelArgs A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    Smem<L>& S = *reinterpret_cast<Smem<L>*>(smem_raw);
    using CF = Cfg<L>;
    constexpr int QP = CF::QP, SP = CF::SP, NB = CF::NB, DB = CF::DB, DT = CF::DT, NDB = CF::NDB;
    constexpr int NT_S = NB * (NB + 1) / 2;          // causal 16x16 tiles of S^T
    constexpr int MAXT = (NT_S + kWaves - 1) / kWaves;
    constexpr int NTT = L / 16;                       // 16-wide tau tiles
    constexpr int NKS = L / 32;                       // k steps of 32 along the chunk
    constexpr int NCT = kDQK / 16;                    // 16-row tiles of this wave's C slice
    constexpr int NUT = (DB / 16 + kWaves - 1) / kWaves;   // 16-col n-update tiles per wave per block

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4;  // k group of the 16x16x32 operands, also the transpose-read group
    const int l16 = lane & 15;
    constexpr int DH = CF::DH, VT = CF::VT, NVG = CF::NVG;
    constexpr int NQ = DT / DH;                 // this wave's 16-row C tiles per d block
    const int vg = wave % NVG;                  // column group
    const int dh = wave / NVG;                  // d partition: tiles dt = q DH + dh of every d block
    auto vcol = [&](int vt) { return 16 * (vg * VT + vt); };   // first column of v tile vt
    // d row of element j of accumulator tile t (see the entry state)
    auto cdrow = [&](int t, int j) {
        const int q = t % NQ;
        return (t / NQ) * DB + 32 * ((q / 2) * DH + dh) + 8 * g16 + 4 * (q % 2) + j;
    };
    const bool gate_wave = (wave == kGateWave);
    // L = 128: the causal 16x16 tiles (tau block tb, sigma block sb) of S^T go to the waves by sigma
    // block, so that a wave reads the transposed K operand of (i) for one or two sigma blocks only.
    // Waves w and w + 4 share a SIMD and split the nine tiles of the sigma blocks p = w % 4 and 7 - p:
    // wave p takes tau blocks p..p+4 of block p (slots 0..4); wave p + 4 takes tau blocks p+5..7 of
    // block p (group A, slots 0..2-p) and tau blocks 7-p..7 of block 7 - p (group B, slot 3 - j for
    // tau block 7 - p + j): five and four tiles per wave, as in the round robin of L = 64.
    const int pr = wave & 3;
    const int nA = wave < 4 ? 5 : 3 - pr;      // tiles of group A (sigma block pr)
    const int tbA = wave < 4 ? pr : pr + 5;   // its first tau block
    const int nB = wave < 4 ? 0 : pr + 1;     // tiles of group B (sigma block 7 - pr)
    auto tile128 = [&](int i, int& tb, int& sb) -> bool {
        if (i < nA) {
            sb = pr;
            tb = tbA + i;
            return true;
        }
        const int j = 3 - i;
        sb = 7 - pr;
        tb = 7 - pr + j;
        return j >= 0 && j < nB;
    };
    uint16_t* const St = CF::ST_ALIAS ? &S.QK[1][0] : S.St_own;
    // Q n tile of this wave (>= NTT: none): with fewer tau tiles than waves, the waves after
    // the two that hold two S tiles take it
    const int dqt = (NTT < kWaves) ? wave - 2 : wave;
    const bool dq_wave = (dqt >= 0 && dqt < NTT);

    const int wi = work_index();
    const int tile = wi % kNTile;
    const int sg = wi / kNTile;
    const int g = sg % A.G;
    const int s = sg / A.G;
    const int v0 = tile * kDVT;
    const int nc_total = (A.T + L - 1) / L;   // the last chunk may be partial
    const int c_begin = g * A.seg_chunks;
    const int c_end = min(nc_total, c_begin + A.seg_chunks);

    SeqRsrc P;
    // the sequence's rows, written out here rather than through seq_rows: this form keeps the
    // compiler's code for the chunk loop as fast as with contiguous-only addressing
    const int bq = A.nh_magic ? static_cast<int>(__umulhi(static_cast<uint32_t>(s), A.nh_magic)) : s;
    P.q = make_rsrc(A.q + static_cast<int64_t>(s) * A.sq[1] + static_cast<int64_t>(bq) * A.sq[0], seq_span(A.T, A.rq, kDQK));
    P.k = make_rsrc(A.k + static_cast<int64_t>(s) * A.sk[1] + static_cast<int64_t>(bq) * A.sk[0], seq_span(A.T, A.rk, kDQK));
    P.v = make_rsrc(A.v + static_cast<int64_t>(s) * A.sv[1] + static_cast<int64_t>(bq) * A.sv[0], seq_span(A.T, A.rv, kDV));
    P.ig = make_rsrc(A.ipre + static_cast<int64_t>(s) * A.T, static_cast<uint32_t>(A.T) * 4);
    P.fg = make_rsrc(A.fpre + static_cast<int64_t>(s) * A.T, static_cast<uint32_t>(A.T) * 4);
    P.h = make_rsrc(A.h + static_cast<int64_t>(s) * A.T * kDV, static_cast<uint32_t>(A.T) * kDV * 2);

    // ---- entry state ------------------------------------------------------------------------
    // C tiles come in pairs over 32 consecutive d: in pair pp of a d block, tile e (0, 1) holds the d
    // with (d mod 8) / 4 == e.  This wave owns pairs pp = pq DH + dh; Cacc[p NQ + 2 pq + e][vt] lane
    // holds C[p DB + 32 pp + 8 g16 + 4 e + j][vcol(vt) + l16], j = 0..3, so the read-out (iii) finds
    // the 8 d of its k slots contiguous in Q.
    f32x4_t Cacc[NDB * NQ][VT];
    const float* Cin = nullptr;
    const float* nin = nullptr;
    float m_prev;
    if (g == 0) {
        Cin = A.C0 ? A.C0 + static_cast<int64_t>(s) * kDQK * kDV : nullptr;
        nin = A.n0 ? A.n0 + static_cast<int64_t>(s) * kDQK : nullptr;
        m_prev = A.m0 ? A.m0[s] : 0.0f;
    } else {
        MLSTM_CHECK(s < A.S && g * A.R - 1 >= 0 && g * A.R - 1 < A.NS, kDbgChunkMfma);
        const float* slot = A.ws + (static_cast<int64_t>(s) * A.NS + g * A.R - 1) * kSlotFloats;
        Cin = slot;
        nin = slot + kDQK * kDV;
        m_prev = slot[kDQK * kDV + kDQK + 2];
    }
    MLSTM_CHECK(s < A.S, kDbgChunkMfma);
    // L = 64: a segment entry slot is loaded after the first chunk's staging loads, so that their
    // waits do not include it (at L = 128 the early load measured faster)
    const bool slot_entry = (Cin && g > 0);
    if (slot_entry && L == 128) {
#pragma unroll
        for (int t = 0; t < NDB * NQ; ++t)
#pragma unroll
            for (int vt = 0; vt < VT; ++vt)
                Cacc[t][vt] = *reinterpret_cast<const f32x4_t*>(Cin + slot_c4(cdrow(t, 0) / 4, v0 + vcol(vt) + l16));
    } else if (slot_entry) {
    } else if (Cin) {
        // C0: the workgroup's 256 x 128 tile in coalesced 16-byte pieces, staged in LDS (rows of
        // kStageP floats, before the chunk loop uses it) and picked up in the accumulator layout
        float* stage = reinterpret_cast<float*>(smem_raw);
#pragma unroll 4
        for (int i = 0; i < (kDQK * kDVT / 4) / kThreads; ++i) {
            const int f = tid + kThreads * i;
            const int row = f / (kDVT / 4), c4 = f % (kDVT / 4);
            *reinterpret_cast<f32x4_t*>(&stage[row * kStageP + 4 * c4]) =
                *reinterpret_cast<const f32x4_t*>(Cin + static_cast<int64_t>(row) * kDV + v0 + 4 * c4);
        }
        __syncthreads();
#pragma unroll
        for (int t = 0; t < NDB * NQ; ++t)
#pragma unroll
            for (int vt = 0; vt < VT; ++vt)
#pragma unroll
                for (int j = 0; j < 4; ++j) Cacc[t][vt][j] = stage[cdrow(t, j) * kStageP + vcol(vt) + l16];
        __syncthreads();   // the staging area is the LDS of the chunk loop
    } else {
#pragma unroll
        for (int t = 0; t < NDB * NQ; ++t)
#pragma unroll
            for (int vt = 0; vt < VT; ++vt) Cacc[t][vt] = f32x4_t{};
    }
    if (tid < kDQK) {
        const float nv = nin ? nin[tid] : 0.0f;
        S.n[0][tid] = nv;
        const uint16_t hi = f32_to_bf16(nv);
        S.nb[0][0][tid] = hi;
        S.nb[0][1][tid] = f32_to_bf16(nv - bf16_to_f32(hi));
    }
    float s_off = 0.0f;   // C = C_acc * e^{s_off}

    // gate wave state: max state and lazy scale after the last chunk whose gates it computed
    float g_m = m_prev, g_s = 0.0f;
    float gi[2] = {0.f, 0.f}, gf[2] = {0.f, 0.f};

    QKRegs<L> rqk;
    VRegs<L> rv;
    VtPacked<L> pv;   // the next chunk's V^T, packed, until its stores
    if (c_begin < c_end) {
        const int t0 = c_begin * L;
        load_qk<L>(rqk, P, t0, 0, tid, A.rq, A.rk);
        if (gate_wave) {
            load_gates<L>(gi, gf, P, t0, lane);
            gate_phase<L>(S.G[c_begin & 1], gi, gf, g_m, g_s, lane, A.T - t0);
        }
        store_qk<L>(S.QK[0], S.QK[0] + CF::QKE, rqk, tid);
#pragma unroll
        for (int part = 0; part < VRegs<L>::PARTS; ++part) {
            load_v_tr<L>(rv, P, t0, v0, wave, lane, part, A.rv);
            vt_transpose<L>(pv, rv, lane, part);
        }
        __syncthreads();   // the first chunk's gates are visible
        vt_store_scaled<L>(S.Vs[1], pv, S.G[c_begin & 1].wC, wave, lane);
        vt_store_plain<L>(S.Vs[0], pv, wave, lane);
        load_qk<L>(rqk, P, t0, 1, tid, A.rq, A.rk);
    }
    if (slot_entry && L == 64) {
        // a segment entry slot (four rows interleaved): each accumulator tile is one 16-byte load
#pragma unroll
        for (int t = 0; t < NDB * NQ; ++t)
#pragma unroll
            for (int vt = 0; vt < VT; ++vt)
                Cacc[t][vt] = *reinterpret_cast<const f32x4_t*>(Cin + slot_c4(cdrow(t, 0) / 4, v0 + vcol(vt) + l16));
    }

    f32x4_t Nacc[VT][NTT];
    f32x4_t Sacc[MAXT];
    f32x4_t dqacc;

    const int tid_outer = tid;
    for (int c = c_begin; c < c_end; ++c) {
        // L = 128: the lane quantities are re-derived from an opaque copy of the thread index in
        // every chunk.  Otherwise the compiler hoists every lane-dependent address out of the loop
        // and, with the larger accumulator set resident, spills them and reloads them through
        // memory each chunk (a reload waits for every staging load in flight).  At L = 64 the
        // recomputation costs more than it saves.
        int tid = tid_outer;
        if constexpr (L == 128) asm volatile("" : "+v"(tid));
        const int lane = tid & 63;
        const int g16 = lane >> 4;
        const int l16 = lane & 15;
        // transpose-read lane roles inside a 16-lane group (16x16x32 operands)
        const int tr_row = (l16 >> 2) + 8 * g16;   // + 4r + k base
        const int tr_col = 4 * (l16 & 3);           // + m/n base
        const int t0 = c * L;
        const int cur = (c - c_begin) & 1;
        const int par = c & 1;
        const GateBuf<L>& Gc = S.G[par];
        __syncthreads();   // the previous chunk is done; block 0, V and the gates of this chunk are visible
        // block 1 -> set 1 (its readers in the previous chunk, the last d block and S~, are done)
        store_qk<L>(S.QK[1], S.QK[1] + CF::QKE, rqk, tid);
        if constexpr (NDB > 2) load_qk<L>(rqk, P, t0, 2, tid, A.rq, A.rk);
        else if (c + 1 < c_end) load_qk<L>(rqk, P, t0 + L, 0, tid, A.rq, A.rk);
        if (gate_wave && c + 1 < c_end) load_gates<L>(gi, gf, P, t0 + L, lane);
        // this chunk's plain V^T (its readers in the previous chunk are done); the next chunk's V,
        // part 0 now, part k at the barrier that opens d block k + 1
        if (c > c_begin) vt_store_plain<L>(S.Vs[0], pv, wave, lane);
        if (c + 1 < c_end) load_v_tr<L>(rv, P, t0 + L, v0, wave, lane, 0, A.rv);
        const float decay_n = Gc.scal[0];
        const float m_next = Gc.scal[1];
        const float s_new = Gc.scal[2];
        const float c_scale = Gc.scal[3];   // != 1: apply this chunk's decay to C_acc eagerly
        const float* n_old = S.n[cur];
        float* n_new = S.n[cur ^ 1];
        const uint16_t* VtT = S.Vs[0];
        const uint16_t* VwT = S.Vs[1];

#pragma unroll
        for (int vt = 0; vt < VT; ++vt)
#pragma unroll
            for (int T = 0; T < NTT; ++T) Nacc[vt][T] = f32x4_t{};
#pragma unroll
        for (int i = 0; i < MAXT; ++i) Sacc[i] = f32x4_t{};
        dqacc = f32x4_t{};

#pragma unroll
        for (int p = 0; p < NDB; ++p) {
            const uint16_t* Qs = S.QK[p & 1];
            const uint16_t* Ks = S.QK[p & 1] + CF::QKE;   // K rows, or K^T at L = 128
            if (p > 0) {
                __syncthreads();   // block p visible, block p - 1 fully read
                if (p + 1 < NDB) {
                    store_qk<L>(S.QK[(p + 1) & 1], S.QK[(p + 1) & 1] + CF::QKE, rqk, tid);
                    if (p + 2 < NDB) load_qk<L>(rqk, P, t0, p + 2, tid, A.rq, A.rk);
                    else if (c + 1 < c_end) load_qk<L>(rqk, P, t0 + L, 0, tid, A.rq, A.rk);
                } else if (c + 1 < c_end) {
                    // block 0 of the next chunk
                    store_qk<L>(S.QK[0], S.QK[0] + CF::QKE, rqk, tid);
                    load_qk<L>(rqk, P, t0 + L, 1, tid, A.rq, A.rk);
                }
                // the next chunk's V, part p - 1, transposed in registers; part p requested
                if (p <= VRegs<L>::PARTS && c + 1 < c_end) {
                    vt_transpose<L>(pv, rv, lane, p - 1);
                    if (p < VRegs<L>::PARTS) load_v_tr<L>(rv, P, t0 + L, v0, wave, lane, p, A.rv);
                }
            }
            // (i) S^T += K_p Q_p^T on this wave's causal tiles.  K^T staging (L = 128): the A operand
            // (K rows sigma, 8 consecutive d) is two transpose reads of 4 K^T rows x 16 tau
            if constexpr (CF::KT) {
                // per group, the A operands (two transpose reads per k step) are read once
#pragma unroll
                for (int grp = 0; grp < 2; ++grp) {
                    const int sb = grp ? 7 - pr : pr;
                    const int n = grp ? nB : nA;
                    const int tb0 = grp ? 7 - pr : tbA;
                    if (n == 0) continue;
                    u32x4_t a[DB / 32];
#pragma unroll
                    for (int ks = 0; ks < DB / 32; ++ks) {
                        const int d0 = 32 * ks + 8 * g16 + (l16 >> 2);
                        a[ks] = cat(tr_read(&Ks[kt_row(d0) * CF::KTP + 16 * sb + tr_col]),
                                    tr_read(&Ks[kt_row(d0 + 4) * CF::KTP + 16 * sb + tr_col]));
                    }
#pragma unroll
                    for (int j = 0; j < (grp ? 4 : MAXT); ++j) {
                        if (j < n) {
                            const uint16_t* qb = &Qs[(16 * (tb0 + j) + l16) * QP + 8 * g16];
                            f32x4_t& acc = Sacc[grp ? 3 - j : j];
#pragma unroll
                            for (int ks = 0; ks < DB / 32; ++ks)
                                acc = mfma16(a[ks], *reinterpret_cast<const u32x4_t*>(qb + 32 * ks), acc);
                        }
                    }
                }
            } else {
#pragma unroll
                for (int i = 0; i < MAXT; ++i) {
                    const int t = wave + kWaves * i;
                    if (t < NT_S) {
                        int tb = 0, rem = t;
                        while (rem > tb) { rem -= tb + 1; ++tb; }
                        const int sb = rem;
                        const uint16_t* qb = &Qs[(16 * tb + l16) * QP + 8 * g16];
                        const uint16_t* ka = &Ks[(16 * sb + l16) * QP + 8 * g16];
#pragma unroll
                        for (int ks = 0; ks < DB / 32; ++ks)
                            Sacc[i] = mfma16(*reinterpret_cast<const u32x4_t*>(ka + 32 * ks),
                                             *reinterpret_cast<const u32x4_t*>(qb + 32 * ks), Sacc[i]);
                    }
                }
            }
            // Q n_{k-1} over this d block: A = Q rows, B = n as bf16 hi / lo columns
            if (dq_wave) {
                const uint16_t* qa = &Qs[(16 * dqt + l16) * QP + 8 * g16];
                const uint16_t* nbp = &S.nb[cur][l16 & 1][p * DB + 8 * g16];
#pragma unroll
                for (int ks = 0; ks < DB / 32; ++ks) {
                    const u32x4_t nbv = (l16 < 2) ? *reinterpret_cast<const u32x4_t*>(nbp + 32 * ks)
                                                  : u32x4_t{0u, 0u, 0u, 0u};
                    dqacc = mfma16(*reinterpret_cast<const u32x4_t*>(qa + 32 * ks), nbv, dqacc);
                }
            }
            // (iii) N^T += C_p^T Q_p^T over this wave's tile pairs: A from the two C tiles of a
            // pair (rows 4 g16 + j of each), converted to bf16 in registers, is k slot 8 g16 + i
            // = d 32 pp + 8 g16 + i; B = 16 bytes of a Q row, shared by the VT column tiles.
            // C goes in as a bf16 pair hi + lo (lo = C - hi, rounded again), so the read-out sees C
            // to about 2^-16: a single bf16 rounding of the state (2^-9) is what a row whose
            // read-out cancels (|C^T q| much smaller than the terms it sums) would amplify
#pragma unroll
            for (int pt = 0; pt < NQ / 2; ++pt) {
                const int q0 = p * NQ + 2 * pt;
                u32x4_t a[VT], alo[VT];
#pragma unroll
                for (int vt = 0; vt < VT; ++vt) {
                    const f32x4_t& c0 = Cacc[q0][vt];
                    const f32x4_t& c1 = Cacc[q0 + 1][vt];
                    a[vt][0] = pack_bf16x2(c0[0], c0[1]);
                    a[vt][1] = pack_bf16x2(c0[2], c0[3]);
                    a[vt][2] = pack_bf16x2(c1[0], c1[1]);
                    a[vt][3] = pack_bf16x2(c1[2], c1[3]);
                    alo[vt][0] = pack_bf16x2(c0[0] - lo_f32(a[vt][0]), c0[1] - hi_f32(a[vt][0]));
                    alo[vt][1] = pack_bf16x2(c0[2] - lo_f32(a[vt][1]), c0[3] - hi_f32(a[vt][1]));
                    alo[vt][2] = pack_bf16x2(c1[0] - lo_f32(a[vt][2]), c1[1] - hi_f32(a[vt][2]));
                    alo[vt][3] = pack_bf16x2(c1[2] - lo_f32(a[vt][3]), c1[3] - hi_f32(a[vt][3]));
                }
                const int dq0 = 32 * (pt * DH + dh) + 8 * g16;   // within the block
                // the Q operand of the next tau tile is requested before this one's MFMAs are issued
                // (the scheduling fence keeps the compiler from waiting on each read in turn)
                u32x4_t b = *reinterpret_cast<const u32x4_t*>(&Qs[l16 * QP + dq0]);
#pragma unroll
                for (int T = 0; T < NTT; ++T) {
                    u32x4_t bn = b;
                    if (T + 1 < NTT) bn = *reinterpret_cast<const u32x4_t*>(&Qs[(16 * (T + 1) + l16) * QP + dq0]);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int vt = 0; vt < VT; ++vt) {
                        Nacc[vt][T] = mfma16(a[vt], b, Nacc[vt][T]);
                        Nacc[vt][T] = mfma16(alo[vt], b, Nacc[vt][T]);
                    }
                    b = bn;
                }
            }

            // (iv) C_p += K_p^T (w e^{-s} V): A = K read transposed (this wave's d tiles),
            // B = V read transposed and scaled by the C-update key weights in registers (rebuilt
            // per d block: a short live range is worth the extra transposed reads)
            if (c_scale != 1.0f) {
#pragma unroll
                for (int q = 0; q < NQ; ++q)
#pragma unroll
                    for (int vt = 0; vt < VT; ++vt) Cacc[p * NQ + q][vt] *= c_scale;
            }
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                // the K^T operands first: their reads are in flight while the weighted V operand is
                // built (the fence keeps the compiler from sinking them below that VALU work)
                u32x4_t a[NQ];
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    if constexpr (CF::KT) {
                        // row m = l16 of tile (pair q / 2, half q % 2) is d = 32 pp + 8 (m / 4) + 4 (q % 2) + m % 4
                        const int d = 32 * ((q / 2) * DH + dh) + 8 * (l16 >> 2) + 4 * (q % 2) + (l16 & 3);
                        a[q] = *reinterpret_cast<const u32x4_t*>(&Ks[kt_row(d) * CF::KTP + 32 * ks + 8 * g16]);
                    } else {
                        // tile (pair q / 2, half q % 2): columns 32 pp + 8 (l16 & 3) + 4 (q % 2) + 0..3
                        const uint16_t* kb = &Ks[(32 * ks + tr_row) * QP + 32 * ((q / 2) * DH + dh) + 2 * tr_col + 4 * (q % 2)];
                        a[q] = cat(tr_read(kb), tr_read(kb + 4 * QP));
                    }
                }
                if constexpr (L == 64) __builtin_amdgcn_sched_barrier(0);
                // lane (n = column vcol(vt) + l16, k group g16) holds tau = 32 ks + 8 g16 + 0..7
                u32x4_t Vw[VT];
#pragma unroll
                for (int vt = 0; vt < VT; ++vt)
                    Vw[vt] = *reinterpret_cast<const u32x4_t*>(&VwT[(vcol(vt) + l16) * CF::TP + 32 * ks + 8 * g16]);
#pragma unroll
                for (int q = 0; q < NQ; ++q)
#pragma unroll
                    for (int vt = 0; vt < VT; ++vt)
                        Cacc[p * NQ + q][vt] = mfma16(a[q], Vw[vt], Cacc[p * NQ + q][vt]);
            }
            // n_p = decay n_p + K_p^T w: A = w as bf16 hi / lo rows, B = K read transposed
#pragma unroll
            for (int j = 0; j < NUT; ++j) {
                const int ut = wave * NUT + j;   // 16-column tile of this d block
                if (ut >= DB / 16) break;
                f32x4_t nacc = f32x4_t{};
#pragma unroll
                for (int ks = 0; ks < NKS; ++ks) {
                    const u32x4_t wa = (l16 < 2) ? *reinterpret_cast<const u32x4_t*>(&Gc.wb[l16 & 1][32 * ks + 8 * g16])
                                                 : u32x4_t{0u, 0u, 0u, 0u};
                    u32x4_t kt;
                    if constexpr (CF::KT) {
                        kt = *reinterpret_cast<const u32x4_t*>(&Ks[kt_row(16 * ut + l16) * CF::KTP + 32 * ks + 8 * g16]);
                    } else {
                        const uint16_t* kb = &Ks[(32 * ks + tr_row) * QP + 16 * ut + tr_col];
                        kt = cat(tr_read(kb), tr_read(kb + 4 * QP));
                    }
                    nacc = mfma16(wa, kt, nacc);
                }
                // rows 0 and 1 (hi and lo weights) of column l16 sit in lanes 0..15
                if (g16 == 0) {
                    const int d = p * DB + 16 * ut + l16;
                    const float nv = decay_n * n_old[d] + nacc[0] + nacc[1];
                    n_new[d] = nv;
                    const uint16_t hi = f32_to_bf16(nv);
                    S.nb[cur ^ 1][0][d] = hi;
                    S.nb[cur ^ 1][1][d] = f32_to_bf16(nv - bf16_to_f32(hi));
                }
            }
        }

        // gates of the next chunk, one chunk ahead; the other waves wait for them at the next
        // barrier, so the gate wave issues ahead of its SIMD partner meanwhile
        if (gate_wave && c + 1 < c_end) {
            __builtin_amdgcn_s_setprio(1);
            gate_phase<L>(S.G[par ^ 1], gi, gf, g_m, g_s, lane, A.T - (t0 + L));
            __builtin_amdgcn_s_setprio(0);
        }

        // finish Q n: columns 0 and 1 of the 16x16 tile are lanes l16 = 0 and 1
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float other = __shfl_down(dqacc[j], 1, 64);
            if (dq_wave && l16 == 0) S.dq[16 * dqt + 4 * g16 + j] = dqacc[j] + other;
        }
        // DH = 2: hand the partial read-out of the tau tiles the other d partition finishes
        if constexpr (DH == 2) {
#pragma unroll
            for (int vt = 0; vt < VT; ++vt)
#pragma unroll
                for (int T = 0; T < NTT; ++T)
                    if ((T & 1) != dh) {
                        MLSTM_CHECK(((((vg * VT + vt) * NTT + T) * 64 + lane) * 4 + 4) <= static_cast<int>(sizeof(S.X) / 4),
                                    kDbgChunkMfma);
                        *reinterpret_cast<f32x4_t*>(&S.X[(((vg * VT + vt) * NTT + T) * 64 + lane) * 4]) = Nacc[vt][T];
                    }
        }
        if constexpr (CF::ST_ALIAS) __syncthreads();   // the last d block is fully read before S~ overwrites it
        // gate matrix on the S^T tiles -> S~ (bf16, tau-major) and row sums (fp32, before the
        // bf16 rounding); branch-free, one 16-byte read of the four sigma exponents per lane
        if constexpr (L == 128) {
#pragma unroll
            for (int i = 0; i < MAXT; ++i) {
                int tb, sb;
                if (tile128(i, tb, sb)) {
                    const int tau = 16 * tb + l16;
                    const float Mt = Gc.M2[tau];
                    const int Rt = Gc.R[tau];
                    const f32x4_t xs = *reinterpret_cast<const f32x4_t*>(&Gc.x2[16 * sb + 4 * g16]);
                    float vals[4];
                    float rsum = 0.f;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int sig = 16 * sb + 4 * g16 + j;
                        const float val = Sacc[i][j] * kQScale * fast_exp2(xs[j] - Mt);
                        // Rt <= sig <= tau as one unsigned comparison (Rt <= tau always)
                        vals[j] = (static_cast<unsigned>(sig - Rt) <= static_cast<unsigned>(tau - Rt)) ? val : 0.f;
                        rsum += vals[j];
                    }
                    u32x2_t o;
                    o[0] = pack_bf16x2(vals[0], vals[1]);
                    o[1] = pack_bf16x2(vals[2], vals[3]);
                    MLSTM_CHECK(tau < L && 16 * sb + 4 * g16 + 4 <= SP &&
                                    tau * SP + 16 * sb + 4 * g16 + 4 <= (CF::ST_ALIAS ? CF::SETE : L * SP),
                                kDbgChunkMfma);
                    *reinterpret_cast<u32x2_t*>(&St[tau * SP + 16 * sb + 4 * g16]) = o;
                    rsum = sum_rows4(rsum);
                    if (g16 == 0) S.rsum_at(tau, sb) = rsum;
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < MAXT; ++i) {
                const int t = wave + kWaves * i;
                if (t < NT_S) {
                    int tb = 0, rem = t;
                    while (rem > tb) { rem -= tb + 1; ++tb; }
                    const int sb = rem;
                    const int tau = 16 * tb + l16;
                    const float Mt = Gc.M2[tau];
                    const int Rt = Gc.R[tau];
                    const f32x4_t xs = *reinterpret_cast<const f32x4_t*>(&Gc.x2[16 * sb + 4 * g16]);
                    float vals[4];
                    float rsum = 0.f;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int sig = 16 * sb + 4 * g16 + j;
                        const float val = Sacc[i][j] * kQScale * fast_exp2(xs[j] - Mt);
                        // Rt <= sig <= tau as one unsigned comparison (Rt <= tau always)
                        vals[j] = (static_cast<unsigned>(sig - Rt) <= static_cast<unsigned>(tau - Rt)) ? val : 0.f;
                        rsum += vals[j];
                    }
                    u32x2_t o;
                    o[0] = pack_bf16x2(vals[0], vals[1]);
                    o[1] = pack_bf16x2(vals[2], vals[3]);
                    MLSTM_CHECK(tau < L && 16 * sb + 4 * g16 + 4 <= SP &&
                                    tau * SP + 16 * sb + 4 * g16 + 4 <= (CF::ST_ALIAS ? CF::SETE : L * SP),
                                kDbgChunkMfma);
                    *reinterpret_cast<u32x2_t*>(&St[tau * SP + 16 * sb + 4 * g16]) = o;
                    rsum = sum_rows4(rsum);
                    if (g16 == 0) S.rsum_at(tau, sb) = rsum;
                }
            }
        }
        // zero the masked 16x16 tiles (sigma block T+1, tau block T) for even T: the k steps
        // of (ii) are 32 wide
        for (int T = 2 * wave; T < NTT; T += 2 * kWaves) {
            const int tau = 16 * T + l16;
            *reinterpret_cast<u32x2_t*>(&St[tau * SP + 16 * T + 16 + 4 * g16]) = u32x2_t{0u, 0u};
        }
        __syncthreads();
        // the next chunk's scaled V^T (its readers, (iv) of this chunk, are done; the next chunk's
        // weights are visible)
        if (c + 1 < c_end) vt_store_scaled<L>(S.Vs[1], pv, S.G[par ^ 1].wC, wave, lane);
        // (ii) N^T = interC * N^T + V^T S~^T, then h = N^T / max(|den|, floor); with DH = 2 each
        // d partition finishes the tau tiles T with T % 2 == dh, after adding the other's partial
#pragma unroll
        for (int T = 0; T < NTT; ++T) {
            if (DH == 2 && (T & 1) != dh) continue;
            const int tau = 16 * T + l16;
            float den = Gc.interN[tau] * S.dq[tau];
            // the row sums of sigma blocks 0..T (L = 128: in groups of four per 16-byte read)
            if constexpr (L == 128) {
#pragma unroll
                for (int sg = 0; 4 * sg <= T; ++sg) {
                    const f32x4_t r4 = *reinterpret_cast<const f32x4_t*>(&S.rsum_at(tau, 4 * sg));
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (4 * sg + j <= T) den += r4[j];
                }
            } else {
#pragma unroll
                for (int sb = 0; sb <= T; ++sb) den += S.rsum_at(tau, sb);
            }
            const float hv = __builtin_amdgcn_rcpf(fmaxf(fabsf(den), Gc.floorv[tau]));
            const float ic = Gc.interC[tau];
#pragma unroll
            for (int vt = 0; vt < VT; ++vt) {
                f32x4_t acc = Nacc[vt][T];
                if constexpr (DH == 2)
                    acc += *reinterpret_cast<const f32x4_t*>(&S.X[(((vg * VT + vt) * NTT + T) * 64 + lane) * 4]);
                acc *= ic;
#pragma unroll
                for (int ks = 0; ks <= T / 2; ++ks) {
                    MLSTM_CHECK(32 * ks + 8 * g16 + 8 <= SP && vcol(vt) + l16 < kDVT && 32 * ks + 8 * g16 + 8 <= CF::TP,
                                kDbgChunkMfma);
                    const u32x4_t b = *reinterpret_cast<const u32x4_t*>(&St[tau * SP + 32 * ks + 8 * g16]);
                    const u32x4_t va = *reinterpret_cast<const u32x4_t*>(&VtT[(vcol(vt) + l16) * CF::TP + 32 * ks + 8 * g16]);
                    acc = mfma16(va, b, acc);
                }
                u32x2_t o;
                o[0] = pack_bf16x2(acc[0] * hv, acc[1] * hv);
                o[1] = pack_bf16x2(acc[2] * hv, acc[3] * hv);
                if constexpr (L == 128) {
                    // 32-bit offsets into the sequence's h: no 64-bit addresses to keep per tau tile; rows
                    // beyond T (a partial last chunk) fall outside the buffer range and are dropped
                    __builtin_amdgcn_raw_buffer_store_b64(o, P.h,
                                                          static_cast<uint32_t>(tau * kDV + v0 + vcol(vt) + 4 * g16) * 2,
                                                          static_cast<uint32_t>(t0) * (kDV * 2), 0);
                } else if (t0 + tau < A.T) {
                    *reinterpret_cast<u32x2_t*>(A.h + (static_cast<int64_t>(s) * A.T + t0 + tau) * kDV + v0 + vcol(vt) +
                                                4 * g16) = o;
                }
            }
        }
        s_off = s_new;
        m_prev = m_next;
    }
    __syncthreads();

    // ---- exit state ---------------------------------------------------------------------------
    const int nfinal = (c_end - c_begin) & 1;
    float* Cout;
    float* nout;
    float* mout;
    const bool write_nm = (tile == 0);
    if (g != A.G - 1) return;
    Cout = A.CT + static_cast<int64_t>(s) * kDQK * kDV;
    nout = A.nT + static_cast<int64_t>(s) * kDQK;
    mout = A.mT + s;
    const float esc = expf(s_off);
#pragma unroll
    for (int t = 0; t < NDB * NQ; ++t) {
#pragma unroll
        for (int vt = 0; vt < VT; ++vt) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d = cdrow(t, j);
                Cout[static_cast<int64_t>(d) * kDV + v0 + vcol(vt) + l16] = Cacc[t][vt][j] * esc;
            }
        }
    }
    if (write_nm && tid < kDQK) {
        nout[tid] = S.n[nfinal][tid];
        if (tid == 0) mout[0] = m_prev;
    }
}

// ---- local segment states as one weighted contraction ------------------------------------------
//
// From an empty state (C = 0, n = 0, m = -inf) the recurrence of Eq. 2-4 over tokens 1..N unrolls to
// a closed form: with b_t the prefix sums of logsig(f~_t) and x_t = i~_t - b_t,
//   m_N = b_N + X,  X = max_t x_t,   C_N = sum_t w_t k_t v_t^T,  n_N = sum_t w_t k_t,  w_t = exp(x_t - X)
// (every weight is <= 1).  With restarts (f~ = -inf) the prefix sums skip the restart tokens, only
// the tokens from the last restart R on carry weight (X is their maximum), and the sub-segment's
// logsig sum is -inf, so the combine drops whatever state entered it.
// A (sub-)segment's local state is therefore one contraction over its
// tokens, with no chunk recurrence: the gates are scanned once over the whole sub-segment, then
// 64-token tiles of K^T and V^T stream through LDS into the MFMA accumulators.  C and n are the
// same quantities the chunkwise update accumulates (bf16 w V operand, bf16 hi / lo weights for n).
constexpr int kLocTile = 64;                  // tokens per tile
constexpr int kLocMax = 4096;                 // tokens per sub-segment (weights held in LDS)
constexpr int kLocP = kLocTile + 8;           // K^T / V^T row pitch: 144 bytes

struct LocSmem {
    uint16_t Kt[2][kDQK * kLocP];             // K^T[d][tau] of a tile, double-buffered
    uint16_t Vt[2][kDVT * kLocP];             // V^T[v][tau] (this workgroup's 128 columns)
    float w[kLocMax];                         // x_t, then the weights w_t
    uint16_t wb[2][kLocMax];                  // w_t as bf16 hi / lo
    float red[3][kWaves];                     // per-wave scan totals, maxima, last restarts
};
static_assert(sizeof(LocSmem) <= 160 * 1024, "LDS budget");

__device__ __forceinline__ uint32_t bload32(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
// Column item regrouping: r[j] holds columns (c, c + 1) of row j as a bf16 pair; c0 / c1 receive
// column c / c + 1 over rows 0..7, in row order.
__device__ __forceinline__ void regroup(const uint32_t (&r)[8], u32x4_t& c0, u32x4_t& c1) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        c0[i] = __builtin_amdgcn_perm(r[2 * i + 1], r[2 * i], 0x05040100u);   // low halves
        c1[i] = __builtin_amdgcn_perm(r[2 * i + 1], r[2 * i], 0x07060302u);   // high halves
    }
}
// One tile in flight: two K column items (2 d x 8 tau) and one V column item (2 v x 8 tau) per
// thread, each read as eight 4-byte loads so the store side can write whole transposed rows.
struct LocRegs {
    uint32_t k[2][8];
    uint32_t v[8];
};
__device__ __forceinline__ void loc_load(LocRegs& r, const SeqRsrc& R, int t, int v0, int tid, uint32_t rk,
                                         uint32_t rv) {
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int item = tid + it * kThreads;
        const uint32_t vo = (8 * (item / (kDQK / 2))) * rk + 4 * (item % (kDQK / 2));
#pragma unroll
        for (int j = 0; j < 8; ++j) r.k[it][j] = bload32(R.k, vo, static_cast<uint32_t>(t + j) * rk);
    }
    const uint32_t vo = (8 * (tid / (kDVT / 2))) * rv + 4 * (tid % (kDVT / 2));
#pragma unroll
    for (int j = 0; j < 8; ++j) r.v[j] = bload32(R.v, vo, static_cast<uint32_t>(t + j) * rv + v0 * 2);
}
__device__ __forceinline__ void loc_store(uint16_t* Kt, uint16_t* Vt, const LocRegs& r, int tid) {
    u32x4_t c0, c1;
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int item = tid + it * kThreads;
        regroup(r.k[it], c0, c1);
        uint16_t* dst = &Kt[(2 * (item % (kDQK / 2))) * kLocP + 8 * (item / (kDQK / 2))];
        *reinterpret_cast<u32x4_t*>(dst) = c0;
        *reinterpret_cast<u32x4_t*>(dst + kLocP) = c1;
    }
    regroup(r.v, c0, c1);
    uint16_t* dst = &Vt[(2 * (tid % (kDVT / 2))) * kLocP + 8 * (tid / (kDVT / 2))];
    *reinterpret_cast<u32x4_t*>(dst) = c0;
    *reinterpret_cast<u32x4_t*>(dst + kLocP) = c1;
}

struct LocalArgs {
    const uint16_t* k;
    const uint16_t* v;
    uint32_t nh_magic;      // as in ChunkKernelArgs
    int64_t sk[2], sv[2];   // as in ChunkKernelArgs
    uint32_t rk, rv;        // their row strides in bytes
    const float* ipre;
    const float* fpre;
    float* ws;
    int S;             // sequences (B NH)
    int T;
    int NS;            // local slots per sequence: (G - 1) segments x R sub-segments
    int R;             // sub-segments per segment
    int seg_tokens;    // tokens per local segment (a multiple of kLocTile)
};

// One workgroup per (sequence, local segment, sub-segment, dv tile); its slot receives C[:, tile],
// and (dv tile 0) n, m_loc and the segment's logsig sum.  kHiLo: the weighted values w v enter the
// matrix cores as bf16 hi + lo (twice the products; the state to about 2^-17 instead of the 2^-9
// of one rounding per term), for the backward pass, whose gradients can cancel against the state.
// (the LDS footprint allows one workgroup per CU, two waves per SIMD: registers are not worth
// saving for a higher occupancy)
template <bool kHiLo>
__global__ void __launch_bounds__(kThreads, 1) __attribute__((amdgpu_waves_per_eu(2, 2)))
local_state_kernel(LocalArgs A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    LocSmem& S = *reinterpret_cast<LocSmem*>(smem_raw);
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, l16 = lane & 15;
    const int wi = work_index();
    const int tile = wi % kNTile;
    const int rest = wi / kNTile;
    const int sl = rest % A.NS;                 // local slot of the sequence
    const int s = rest / A.NS;
    const int g = sl / A.R, r = sl % A.R;
    const int v0 = tile * kDVT;
    const int ntiles = A.seg_tokens / kLocTile;
    const int tps = (ntiles + A.R - 1) / A.R;
    const int tile_b = min(ntiles, r * tps), tile_e = min(ntiles, tile_b + tps);
    const int tb = g * A.seg_tokens + tile_b * kLocTile;
    const int ntok = (tile_e - tile_b) * kLocTile;

    SeqRsrc P;
    P.k = make_rsrc(seq_rows(A.k, s, A.nh_magic, A.sk), seq_span(A.T, A.rk, kDQK));
    P.v = make_rsrc(seq_rows(A.v, s, A.nh_magic, A.sv), seq_span(A.T, A.rv, kDV));
    P.ig = make_rsrc(A.ipre + static_cast<int64_t>(s) * A.T, static_cast<uint32_t>(A.T) * 4);
    P.fg = make_rsrc(A.fpre + static_cast<int64_t>(s) * A.T, static_cast<uint32_t>(A.T) * 4);

    LocRegs rg;
    if (ntok > 0) loc_load(rg, P, tb, v0, tid, A.rk, A.rv);   // first tile, in flight during the gate pass

    // gates: block-wide prefix sums of logsig(f~) in rounds of 512 tokens (restart tokens add
    // nothing), x_t into LDS, the last restart R, then X over the tokens from R on
    float carry = 0.0f, rmax = -1.0f, xall = -INFINITY;
    for (int j0 = 0; j0 < ntok; j0 += kThreads) {
        const int t = j0 + tid;
        const bool valid = t < ntok;
        const float fv = valid ? bloadf(P.fg, 4 * t, 4 * tb) : 0.0f;
        const float iv = valid ? bloadf(P.ig, 4 * t, 4 * tb) : 0.0f;
        const float lg = valid ? flogsig(fv) : 0.0f;
        const bool rs = (lg == -INFINITY);
        if (rs) rmax = static_cast<float>(t);
        const float incl = wave_incl_sum(rs ? 0.0f : lg);
        if (lane == 63) S.red[0][wave] = incl;
        __syncthreads();
        float before = carry, total = 0.0f;
#pragma unroll
        for (int w2 = 0; w2 < kWaves; ++w2) {
            const float tw = S.red[0][w2];
            if (w2 < wave) before += tw;
            total += tw;
        }
        carry += total;
        const float x = valid ? iv - (before + incl) : -INFINITY;
        if (valid) S.w[t] = x;
        xall = fmaxf(xall, x);
        __syncthreads();   // red[0] is rewritten by the next round
    }
    const float wr = lane63(wave_incl_max(rmax));
    if (lane == 0) S.red[2][wave] = wr;
    __syncthreads();   // the x_t and the restarts of every wave are visible
    float Rf = -1.0f;
#pragma unroll
    for (int w2 = 0; w2 < kWaves; ++w2) Rf = fmaxf(Rf, S.red[2][w2]);
    const int Rl = static_cast<int>(Rf);   // last restart of the sub-segment, -1: none
    float xmax = xall;   // no restart: the maximum over every token
    if (Rl >= 0) {       // block-uniform: only the tokens from the restart on
        xmax = -INFINITY;
        for (int t = Rl + tid; t < ntok; t += kThreads) xmax = fmaxf(xmax, S.w[t]);
    }
    const float wm = lane63(wave_incl_max(xmax));
    if (lane == 0) S.red[1][wave] = wm;
    __syncthreads();
    float X = -INFINITY;
#pragma unroll
    for (int w2 = 0; w2 < kWaves; ++w2) X = fmaxf(X, S.red[1][w2]);
    for (int t = tid; t < ntok; t += kThreads) {
        const float wv = (t < Rl || X == -INFINITY) ? 0.0f : fexp(S.w[t] - X);
        S.w[t] = wv;
        const uint16_t hi = f32_to_bf16(wv);
        S.wb[0][t] = hi;
        S.wb[1][t] = f32_to_bf16(wv - bf16_to_f32(hi));
    }

    // contraction: wave (dh, vg) owns C[128 dh + 0..127][32 vg + 0..31] as 8 x 2 tiles; it also
    // accumulates n over its d tiles 2 vg and 2 vg + 1
    const int dh = wave >> 2, vg = wave & 3;
    f32x4_t Cacc[8][2];
    f32x4_t nacc[2];
#pragma unroll
    for (int q = 0; q < 8; ++q) Cacc[q][0] = Cacc[q][1] = f32x4_t{};
    nacc[0] = nacc[1] = f32x4_t{};
    const int nt = ntok / kLocTile;
    if (nt > 0) {
        loc_store(S.Kt[0], S.Vt[0], rg, tid);
        if (nt > 1) loc_load(rg, P, tb + kLocTile, v0, tid, A.rk, A.rv);
    }
    for (int i = 0; i < nt; ++i) {
        __syncthreads();   // tile i and the weights are visible; the other buffer's readers are done
        if (i + 1 < nt) {
            loc_store(S.Kt[(i + 1) & 1], S.Vt[(i + 1) & 1], rg, tid);
            if (i + 2 < nt) loc_load(rg, P, tb + (i + 2) * kLocTile, v0, tid, A.rk, A.rv);
        }
        const uint16_t* Kt = S.Kt[i & 1];
        const uint16_t* Vt = S.Vt[i & 1];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int t0 = i * kLocTile + 32 * ks + 8 * g16;   // this lane's 8 k slots
            const f32x4_t wa0 = *reinterpret_cast<const f32x4_t*>(&S.w[t0]);
            const f32x4_t wa1 = *reinterpret_cast<const f32x4_t*>(&S.w[t0 + 4]);
            const float wv[8] = {wa0[0], wa0[1], wa0[2], wa0[3], wa1[0], wa1[1], wa1[2], wa1[3]};
            u32x4_t Vw[2], Vl[2];
#pragma unroll
            for (int vt = 0; vt < 2; ++vt) {
                const u32x4_t raw = *reinterpret_cast<const u32x4_t*>(&Vt[(32 * vg + 16 * vt + l16) * kLocP + 32 * ks + 8 * g16]);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float x0 = lo_f32(raw[u]) * wv[2 * u], x1 = hi_f32(raw[u]) * wv[2 * u + 1];
                    Vw[vt][u] = pack_bf16x2(x0, x1);
                    if constexpr (kHiLo) Vl[vt][u] = pack_bf16x2(x0 - lo_f32(Vw[vt][u]), x1 - hi_f32(Vw[vt][u]));
                }
            }
            const uint16_t* kb = &Kt[(128 * dh + l16) * kLocP + 32 * ks + 8 * g16];
            u32x4_t a[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) a[q] = *reinterpret_cast<const u32x4_t*>(kb + 16 * q * kLocP);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                Cacc[q][0] = mfma16(a[q], Vw[0], Cacc[q][0]);
                Cacc[q][1] = mfma16(a[q], Vw[1], Cacc[q][1]);
                if constexpr (kHiLo) {
                    Cacc[q][0] = mfma16(a[q], Vl[0], Cacc[q][0]);
                    Cacc[q][1] = mfma16(a[q], Vl[1], Cacc[q][1]);
                }
            }
            // n over d tiles 2 vg and 2 vg + 1 (rows re-read by address: no wave-dependent branch)
            const u32x4_t wa = (l16 < 2) ? *reinterpret_cast<const u32x4_t*>(&S.wb[l16 & 1][t0]) : u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
            for (int e = 0; e < 2; ++e)
                nacc[e] = mfma16(wa, *reinterpret_cast<const u32x4_t*>(kb + 16 * (2 * vg + e) * kLocP), nacc[e]);
        }
    }

    // slot (s, local slot sl): C [DQK x DV] row-major, then n, m_loc, logsig sum
    MLSTM_CHECK(s < A.S && sl < A.NS && ntok <= kLocMax, kDbgChunkMfma);
    float* slot = A.ws + (static_cast<int64_t>(s) * A.NS + sl) * kSlotFloats;
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
        for (int vt = 0; vt < 2; ++vt)
            *reinterpret_cast<f32x4_t*>(slot + slot_c4(32 * dh + 4 * q + g16, v0 + 32 * vg + 16 * vt + l16)) = Cacc[q][vt];
    if (tile == 0) {
        if (g16 == 0) {
#pragma unroll
            for (int e = 0; e < 2; ++e) slot[kDQK * kDV + 128 * dh + 16 * (2 * vg + e) + l16] = nacc[e][0] + nacc[e][1];
        }
        if (tid == 0) {
            slot[kDQK * kDV + kDQK] = carry + X;      // m_loc (-inf for an empty sub-segment)
            slot[kDQK * kDV + kDQK + 1] = Rl >= 0 ? -INFINITY : carry;   // sum of logsig(f~)
        }
    }
}

// Running entry states from the local (sub-)segment states, in place: the last slot of segment g
// (slot g R + R - 1) receives the state after local slots 0..g R + R - 1, the entry state of
// segment g + 1; the other sub-segment slots are only read.
__global__ void __launch_bounds__(256) combine_kernel(float* ws, const float* C0, const float* n0, const float* m0,
                                                      int NS, int R) {
    const int s = blockIdx.y;
    float* base = ws + static_cast<int64_t>(s) * NS * kSlotFloats;
    // scalar chain of entry max states (every block computes it; block 0 stores it)
    float m_in = m0 ? m0[s] : 0.0f;
    constexpr int kE4 = (kDQK * kDV + kDQK) / 4;
    const int e4 = blockIdx.x * blockDim.x + threadIdx.x;
    float4 cur = make_float4(0.f, 0.f, 0.f, 0.f);
    if (e4 < kE4) {
        if (e4 < kDQK * kDV / 4) {
            if (C0) {
                // slot float4 e4 holds rows 4 (e4 / DV) + 0..3 of column e4 % DV; C0 is row-major
                const float* c0 = C0 + static_cast<int64_t>(s) * kDQK * kDV + static_cast<int64_t>(4 * (e4 / kDV)) * kDV + e4 % kDV;
                cur = make_float4(c0[0], c0[kDV], c0[2 * kDV], c0[3 * kDV]);
            }
        } else if (n0) {
            cur = reinterpret_cast<const float4*>(n0 + static_cast<int64_t>(s) * kDQK)[e4 - kDQK * kDV / 4];
        }
    }
    // slots in batches: all loads of a batch are issued before its dependent chain of updates
    constexpr int kBatch = 8;
    for (int g0 = 0; g0 < NS; g0 += kBatch) {
        const int nbat = min(kBatch, NS - g0);
        float4 loc[kBatch];
        float mloc[kBatch], gs[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (u < nbat) {
                const float* slot = base + static_cast<int64_t>(g0 + u) * kSlotFloats;
                mloc[u] = slot[kDQK * kDV + kDQK];
                gs[u] = slot[kDQK * kDV + kDQK + 1];
                if (e4 < kE4) loc[u] = reinterpret_cast<const float4*>(slot)[e4];
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (u < nbat) {
                float* slot = base + static_cast<int64_t>(g0 + u) * kSlotFloats;
                // a restart inside the slot (gs = -inf) drops the running state; an empty slot
                // (m_loc = -inf) adds nothing
                const float carried = gs[u] + m_in;
                const float m_new = fmaxf(carried, mloc[u]);
                const float a = (carried == -INFINITY) ? 0.0f : expf(carried - m_new);
                const float b = (mloc[u] == -INFINITY) ? 0.0f : expf(mloc[u] - m_new);
                const bool entry = ((g0 + u) % R) == R - 1;
                if (e4 < kE4) {
                    cur.x = a * cur.x + b * loc[u].x;
                    cur.y = a * cur.y + b * loc[u].y;
                    cur.z = a * cur.z + b * loc[u].z;
                    cur.w = a * cur.w + b * loc[u].w;
                    if (entry) reinterpret_cast<float4*>(slot)[e4] = cur;
                }
                if (entry && blockIdx.x == 0 && threadIdx.x == 0) slot[kDQK * kDV + kDQK + 2] = m_new;
                m_in = m_new;
            }
        }
    }
}

// q, k, v strides of a call: the caller's (elements; batch, head, token for each), or contiguous
// [B, NH, T, D] rows; the kernels take {batch - NH head, head} per matrix (see seq_rows)
void set_strides(const ChunkArgs& a, uint32_t& nh_magic, int64_t* sq, int64_t* sk, int64_t* sv, uint32_t* rq,
                 uint32_t* rk, uint32_t* rv) {
    nh_magic = a.NH > 1 ? static_cast<uint32_t>((uint64_t(1) << 32) / static_cast<uint64_t>(a.NH) + 1) : 0u;
    const int64_t T = a.T, NH = a.NH;
    const int64_t st[9] = {NH * T * kDQK, T * kDQK, kDQK, NH * T * kDQK, T * kDQK, kDQK, NH * T * kDV, T * kDV, kDV};
    const int64_t* x = a.strides ? a.strides : st;
    if (sq) {
        sq[0] = x[0] - NH * x[1];
        sq[1] = x[1];
    }
    sk[0] = x[3] - NH * x[4];
    sk[1] = x[4];
    sv[0] = x[6] - NH * x[7];
    sv[1] = x[7];
    if (rq) *rq = static_cast<uint32_t>(x[2] * 2);
    *rk = static_cast<uint32_t>(x[5] * 2);
    *rv = static_cast<uint32_t>(x[8] * 2);
}

template <int L>
hipError_t launch_variant(const ChunkKernelArgs& a, int S, hipStream_t stream) {
    const size_t lds = sizeof(Smem<L>);
    auto kern = chunk_mfma_kernel<L>;
    static std::atomic<uint64_t> raised{0};
    hipError_t e = raise_dynamic_lds(reinterpret_cast<const void*>(kern), lds, raised);
    if (e != hipSuccess) return e;
    const dim3 grid(static_cast<unsigned>(S * a.G * kNTile));
    hipLaunchKernelGGL(kern, grid, dim3(kThreads), lds, stream, a);
    return hipGetLastError();
}

hipError_t launch_local(const LocalArgs& a, int S, hipStream_t stream, bool hilo = false) {
    const size_t lds = sizeof(LocSmem);
    static std::atomic<uint64_t> raised[2]{{0}, {0}};
    auto kern = hilo ? local_state_kernel<true> : local_state_kernel<false>;
    hipError_t e = raise_dynamic_lds(reinterpret_cast<const void*>(kern), lds, raised[hilo ? 1 : 0]);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(S * a.NS * kNTile)), dim3(kThreads), lds, stream, a);
    return hipGetLastError();
}

// sub-segments of a local segment: at most kLocMax tokens each
int local_subsegments(int seg_tokens) { return (seg_tokens + kLocMax - 1) / kLocMax; }

}  // namespace

bool chunk_mfma_supported(mlstm_dtype dt, int DQK, int DV, int L) {
    return dt == MLSTM_BF16 && DQK == kDQK && DV == kDV && (L == 64 || L == 128);
}

int chunk_mfma_segments(int B, int NH, int T, int L) {
    const int S = B * NH;
    const int nc = (T + L - 1) / L;
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
    const int nc = (T + L - 1) / L;
    const int seg_tokens = ((nc + G - 1) / G) * L;
    return static_cast<size_t>(B) * NH * (G - 1) * local_subsegments(seg_tokens) * kSlotFloats * sizeof(float);
}

// ---- the segment schedule ---------------------------------------------------------------------
SegmentShape segment_shape(int B, int NH, int T, int L, bool use_segments) {
    SegmentShape sh{};
    const int nc = (T + L - 1) / L;
    sh.G = (use_segments && nc > 0) ? chunk_mfma_segments(B, NH, T, L) : 1;
    sh.seg_chunks = sh.G > 1 ? (nc + sh.G - 1) / sh.G : nc;
    sh.R = sh.G > 1 ? local_subsegments(sh.seg_chunks * L) : 1;
    return sh;
}

hipError_t launch_segment_states(const ChunkArgs& a, int L, const SegmentShape& sh, float* seg, bool hilo,
                                 hipStream_t stream) {
    if (sh.G <= 1) return hipSuccess;
    const int S = a.B * a.NH;
    LocalArgs la{};
    la.k = static_cast<const uint16_t*>(a.k);
    la.v = static_cast<const uint16_t*>(a.v);
    set_strides(a, la.nh_magic, nullptr, la.sk, la.sv, nullptr, &la.rk, &la.rv);
    la.ipre = a.ipre;
    la.fpre = a.fpre;
    la.ws = seg;
    la.S = S;
    la.T = a.T;
    la.NS = (sh.G - 1) * sh.R;
    la.R = sh.R;
    la.seg_tokens = sh.seg_chunks * L;
    hipError_t e = launch_local(la, S, stream, hilo);
    if (e != hipSuccess) return e;
    constexpr int kE4 = (kDQK * kDV + kDQK) / 4;
    hipLaunchKernelGGL(combine_kernel, dim3((kE4 + 255) / 256, S), dim3(256), 0, stream, seg, a.C0, a.n0, a.m0, la.NS,
                       sh.R);
    return hipGetLastError();
}

hipError_t launch_chunk_mfma(const ChunkArgs& a, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    const int S = a.B * a.NH;
    const bool use_segments =
        workspace != nullptr && workspace_bytes >= chunk_mfma_workspace_bytes(a.B, a.NH, a.T, a.DQK, a.DV, a.L);
    const SegmentShape sh = segment_shape(a.B, a.NH, a.T, a.L, use_segments);

    ChunkKernelArgs k{};
    k.q = static_cast<const uint16_t*>(a.q);
    k.k = static_cast<const uint16_t*>(a.k);
    k.v = static_cast<const uint16_t*>(a.v);
    set_strides(a, k.nh_magic, k.sq, k.sk, k.sv, &k.rq, &k.rk, &k.rv);
    k.ipre = a.ipre;
    k.fpre = a.fpre;
    k.C0 = a.C0;
    k.n0 = a.n0;
    k.m0 = a.m0;
    k.ws = static_cast<float*>(workspace);
    k.S = S;
    k.T = a.T;
    k.G = sh.G;
    k.R = sh.R;
    k.NS = (sh.G - 1) * sh.R;
    k.seg_chunks = sh.seg_chunks;
    k.h = static_cast<uint16_t*>(a.h);
    k.CT = a.CT;
    k.nT = a.nT;
    k.mT = a.mT;

    hipError_t e = launch_segment_states(a, a.L, sh, k.ws, false, stream);
    if (e != hipSuccess) return e;
    return (a.L == 64) ? launch_variant<64>(k, S, stream) : launch_variant<128>(k, S, stream);
}

// ---- fixed scratch for callers that cannot allocate ---------------------------------------------
// The segment slots of mlstm_chunkwise_fwd_noalloc.  Every slot a call reads is written earlier in
// the same call (local pass, then combine), so nothing needs clearing between calls; calls that
// overlap on one device share this array and race.
namespace {
__device__ __attribute__((aligned(256))) unsigned char scratch[kChunkScratchBytes];
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};
}  // namespace

hipError_t chunk_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        // the device address of this device's copy (the host-side name is not a device address)
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_chunk_mfma)
#endif

}  // namespace mlstm
