// Chunkwise backward of the mLSTM cell on bf16 MFMA for the xLSTM 7B head shape
// (DQK = 256, DV = 512), chunk length 64: the gradients of sum(h~ . dh) with respect to
// q, k, v, the gate pre-activations and the initial state (C0, n0, m0).
//
// Math.  Per chunk c with entry state (C, n, m_prev) (stabilised by m_prev), the gates of the
// forward (in-chunk prefix sums b, x = i~ - b, last restart R_tau, M_tau, key weights
// w_tau = exp(x_tau - M_L), decay = exp(m_prev - M_L)), g_tau = exp(m_prev - M_tau) and
// floor_tau = exp(-(b_tau + M_tau)) (App. D.1), with q^ = q / sqrt(DQK):
//
//   S = Q^ K^T,  E_ts = exp(x_s - M_t) for R_t <= s <= t (else 0),  St = S o E
//   D_t = g_t (q^_t . n) + sum_s St_ts,  den_t = max(|D_t|, floor_t),  h~_t = N_t / den_t with
//   N_t = g_t (C^T q^_t) + sum_s St_ts v_s
//   U = dH / den (rows),  w_t = -(dh_t . N_t) sign(D_t) / den_t^2  where |D_t| > floor_t, else 0
//   P = E o (U V^T + w 1^T)
//   dq^ = P K + diag(g) (U C^T + w n^T),   dk = P^T Q^ + diag(wkey) (V Gam^T + 1 gam^T),
//   dv  = St^T U + diag(wkey) K Gam,
// where (Gam_c, gam_c) is the gradient reaching chunk c's exit state (C_c, n_c), in the units of
// its stabiliser, from all later chunks; it runs backwards through the state recurrence of
// Eqs. 3-4 in chunk form:
//   Gam_{c-1} = decay_c Gam_c + L_c,   L_c = Q^T diag(g / den) dH,
//   gam_{c-1} = decay_c gam_c + z_c,   z_c = Q^T (g o w) / sqrt(DQK)
// (Gam of the last chunk is zero; Gam_{-1}, gam_{-1} are the gradients of C0 and n0, and
// dm0 = <Gam_{-1}, C0> + gam_{-1} . n0 since the unstabilised state is e^{m0} (C0, n0)).
// The gate gradients follow from the two row sums r_t = q_t . dq_t and c_t = k_t . dk_t:
//   di~_t = c_t,  dlogsig(f~_t) = sum_{t' >= t} (r_t' - c_t'),  df~_t = that times sigmoid(-f~_t)
// (a forget gate of zero, f~ = -inf, is a restart; its own gradient is zero).
//
// dh_t . N_t is formed in fp32 from its two parts, g_t q^_t . (C dh_t) and sum_s St_ts (dh_t . v_s),
// rather than from the forward's rounded h~: where the two terms of dq nearly cancel, the bf16
// rounding of h~ would dominate the result.  The forward's output is not an input.
//
// Passes (one stream, in order):
//   walk    the prefill's segment schedule (local pass in the bf16 hi + lo form, combine) for the
//           entry states of segments of several chunks, then a walk over each segment's chunks per
//           dv tile, holding its slice of the state in registers: per chunk the tile's partial sum of
//           X = dH C^T on the entry state, its share of q^_t . X_t, then the state update; n and m
//           entering each chunk go to its slot
//   xsum    X, the sum of the four tiles' partials, into dq
//   intra   one workgroup per chunk: gates, S, D, den; per 128-column piece of dv, (dH V^T), the
//           intra term of dv and the piece's columns of L_c; then w, P, dq (complete), the intra
//           term of dk and z_c; writes the key weights, the chunk's decay and q_t . dq_t
//   scan    the reverse recurrence of (Gam, gam), elementwise over the state (fp32), writing Gam_c
//           rounded once to bf16; dC0, dn0 and partial sums of dm0
//   interkv one workgroup per chunk: the inter terms of dk and dv from Gam_c, read once; k . dk
//   gates   one workgroup per sequence: the reverse prefix sums of r - c, di~ and df~, dm0
//
// MFMA mapping (16x16x32 bf16, fp32 accumulate): lane (l16, g16) holds A[m = l16][k = 8 g16 + 0..7]
// and B[k = 8 g16 + 0..7][n = l16] and receives D[m = 4 g16 + 0..3][n = l16].  An operand whose
// contraction index is contiguous in memory is one 16-byte row read; otherwise it comes from a
// row-major [k][n] tile in LDS through the transpose read.  Every product is arranged so that its
// output lane holds four consecutive elements of one output row (one 16-byte store).
//
// Rows past the end of the sequence (a partial last chunk) are read through buffer resources with
// the row offset in the range-checked offset, so they read as zero.
#include "chunk_common.h"
#include "launch.h"

namespace mlstm {
namespace {

constexpr int kBL = 64;                                   // tokens per chunk
constexpr int kBT = 256;                                  // threads per workgroup (4 waves)
constexpr int kQP = kDQK + 8;                             // LDS pitch of Q, K rows (528 bytes)
constexpr int kPP = kBL + 8;                              // LDS pitch of [tau][sigma] tiles (144 bytes)
constexpr int kWP = 128 + 8;                              // LDS pitch of 128-column pieces (272 bytes)
constexpr int kHP = kDV + 8;                              // LDS pitch of full dv rows (1040 bytes)
constexpr int64_t kCV = static_cast<int64_t>(kDQK) * kDV; // elements of one state matrix
constexpr int64_t kLzFloats = kCV + kDQK;                 // L_c then z_c
constexpr int kScanE4 = static_cast<int>(kLzFloats / 4);  // float4 items of the reverse scan
constexpr int kScanBlocks = (kScanE4 + 255) / 256;
constexpr int kTokF = 1;                                  // per-token floats: the key weight
constexpr int kPartF = 8;                                 // per-token partial sums: q^.X x 4 (then q.dq), k.dk x 4

struct BwdParams {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const uint16_t* dh;
    const float* ipre;
    const float* fpre;
    const float* C0;     // NULL: zero initial state (with n0, m0)
    const float* n0;
    const float* m0;
    float* dq;
    float* dk;
    float* dv;
    float* dip;
    float* dfp;
    float* dC0;          // NULL: not requested (with dn0, dm0)
    float* dn0;
    float* dm0;
    float* slots;        // S (NC - 1) slots: n, m entering chunk c in slot c - 1, then L_c, z_c
    uint16_t* hl;        // S (NC - 1) x DQK x DV: Gam_c in bf16
    float* lz0;          // S x (DQK DV + DQK): L_0, z_0
    float* gamn;         // S x NC x DQK: gam_c
    float* tok;          // S x T x kTokF
    float* part;         // S x T x kPartF
    float* chunk;        // S x NC: decay of each chunk
    float* dmp;          // S x kScanBlocks: partial sums of dm0
    int T;
    int NC;
};

__device__ __forceinline__ float* lz_of(const BwdParams& A, int s, int c) {
    MLSTM_CHECK(c >= 0 && c < A.NC && s >= 0, kDbgChunkBwd);
    return c ? A.slots + (static_cast<int64_t>(s) * (A.NC - 1) + c - 1) * kSlotFloats
             : A.lz0 + static_cast<int64_t>(s) * kLzFloats;
}
__device__ __forceinline__ uint16_t* hl_of(const BwdParams& A, int s, int slot) {
    MLSTM_CHECK(slot >= 0 && slot < A.NC - 1 && s >= 0, kDbgChunkBwd);
    return A.hl + (static_cast<int64_t>(s) * (A.NC - 1) + slot) * kCV;
}

__device__ __forceinline__ u32x4_t lds16(const uint16_t* p) { return *reinterpret_cast<const u32x4_t*>(p); }
__device__ __forceinline__ u32x2_t lds_u32x2(const uint16_t* p) { return *reinterpret_cast<const u32x2_t*>(p); }
// operand whose contraction index runs along LDS rows: lane gets row r0 + l16, k = k0 + 8 g16 + 0..7
__device__ __forceinline__ u32x4_t row_op(const uint16_t* base, int pitch, int r0, int k0, int lane) {
    return lds16(base + (r0 + (lane & 15)) * pitch + k0 + 8 * (lane >> 4));
}
// operand from a row-major [k][n] LDS tile: lane gets column n0 + l16, k = k0 + 8 g16 + 0..7
__device__ __forceinline__ u32x4_t tr_op(const uint16_t* base, int pitch, int k0, int n0, int lane) {
    const int g16 = lane >> 4, l16 = lane & 15;
    const uint16_t* p = base + (k0 + 8 * g16 + (l16 >> 2)) * pitch + n0 + 4 * (l16 & 3);
    return cat(tr_read(p), tr_read(p + 4 * pitch));
}
__device__ __forceinline__ float bf_at(const u32x4_t& w, int e) {
    return (e & 1) ? hi_f32(w[e >> 1]) : lo_f32(w[e >> 1]);
}
// fp32 -> bf16 hi + lo parts of 8 values, packed as two MFMA operands
__device__ __forceinline__ void split8(const float4& a, const float4& b, u32x4_t& hi, u32x4_t& lo) {
    const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        hi[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
        lo[i] = pack_bf16x2(x[2 * i] - lo_f32(hi[i]), x[2 * i + 1] - hi_f32(hi[i]));
    }
}
__device__ __forceinline__ float wave_total(float x) { return lane63(wave_incl_sum(x)); }

// rows t0 .. t0 + 63, columns col0 .. col0 + NCOL - 1 of a [T][row_elems] bf16 matrix into LDS
template <int NCOL>
__device__ __forceinline__ void stage_rows(uint16_t* dst, int pitch, __amdgpu_buffer_rsrc_t r, int row_elems, int t0,
                                           int col0, int tid) {
    constexpr int PPR = NCOL / 8, N = kBL * PPR / kBT;
    u32x4_t tmp[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int e = tid + kBT * i, row = e / PPR, pc = e % PPR;
        tmp[i] = bload128(r, static_cast<uint32_t>((t0 + row) * row_elems + col0 + 8 * pc) * 2u, 0);
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int e = tid + kBT * i, row = e / PPR, pc = e % PPR;
        *reinterpret_cast<u32x4_t*>(dst + row * pitch + 8 * pc) = tmp[i];
    }
}

// ---- gates of one chunk (one wave, lane = row) -------------------------------------------------
struct BGate {
    float x, M, g, fl, wk;
    int R;
};
__device__ __forceinline__ void bwd_gates(__amdgpu_buffer_rsrc_t ig, __amdgpu_buffer_rsrc_t fg, int T, int t0,
                                          float m_prev, int lane, BGate& G, float& decay) {
    const int t = t0 + lane;
    const bool ok = t < T;
    const uint32_t off = static_cast<uint32_t>(t) * 4u;
    const float fv = bloadf(fg, off, 0), iv = bloadf(ig, off, 0);
    const float lg = ok ? flogsig(fv) : 0.0f;
    const bool rs = (lg == -INFINITY);
    const bool any = __builtin_amdgcn_ballot_w64(rs) != 0;
    const float b = wave_incl_sum(rs ? 0.0f : lg);
    const float x = ok ? iv - b : -INFINITY;
    float r = -1.0f, p;
    if (any) {
        r = wave_incl_max(rs ? static_cast<float>(lane) : -1.0f);
        p = wave_seg_incl_max(x, rs);
    } else {
        p = wave_incl_max(x);
    }
    const float pL = lane63(p), rL = lane63(r);
    const bool restart = rL >= 0.0f;
    const float ML = restart ? pL : fmaxf(m_prev, pL);
    const bool fresh = r >= 0.0f;
    const float M = fresh ? p : fmaxf(m_prev, p);
    G.x = x;
    G.M = M;
    G.R = static_cast<int>(r);
    G.g = (fresh || M == -INFINITY) ? 0.0f : fexp(m_prev - M);
    G.fl = fexp(-(b + M));
    const bool none = (x == -INFINITY) || (static_cast<float>(lane) < rL);
    G.wk = none ? 0.0f : fexp(x - ML);
    decay = (restart || ML == -INFINITY || m_prev == -INFINITY) ? 0.0f : fexp(m_prev - ML);
}

// ---- the backward's forward walk ----------------------------------------------------------------
// The backward needs, for every 64-token chunk c, X_c = dH_c C_c^T on the state C_c entering the chunk
// (the inter-chunk term of dq), with q^_t . X_t, and the chunk's entry normaliser and max state.  A
// walk over the chunks gives them without writing the states out: one workgroup of 8 waves per
// (sequence, 128-column dv tile, segment), with the gate phase and lazy scale of chunk_mfma_kernel<64>,
// holds its 256 x 128 slice of C in registers and per chunk
//   - forms X^T = C dH^T over its 128 columns (the four tiles' partial sums are added by the
//     backward) and its share of q^ . X,
//   - applies the update C += K^T (w e^{-s} V), the weighted values as a bf16 pair hi + lo (products
//     to about 2^-17 rather than the 2^-9 of one rounding, because the backward's gradients can
//     cancel against the state), and n += K^T w,
//   - writes n and m entering the chunk into slot c - 1 (tile 0).
// Layout: wave w owns d = 32 w + 0..31 (two 16-column tiles dt) and all 128 v, as accumulator tiles
// of C^T: tile (dt, pp, e) lane (l16, g16) holds C[32 w + 16 dt + l16][32 pp + 8 g16 + 4 e + j],
// j = 0..3.  The two tiles e of a pair give a lane eight consecutive v, the A operand of C dH^T (with
// 16-byte reads of dH rows); the update reads the weighted V^T rows in the same permuted order.
// Segment g >= 1 enters from the segment slots of the local pass (in its hi + lo form) and the
// combine.
constexpr int kWalkHP = kDVT + 8;   // dH row pitch (elements): 272 bytes
struct WalkSmem {
    uint16_t K[Cfg<64>::NDB][64 * Cfg<64>::QP];   // the chunk's K rows, two d blocks of 128
    uint16_t Vw[2][kDVT * Cfg<64>::TP];           // (w e^{-s} V)^T of the chunk as bf16 hi [0] and lo [1]
    uint16_t dH[64 * kWalkHP];                     // the chunk's dH rows, this tile's 128 columns
    float n[2][kDQK];                              // fp32 normaliser, double-buffered across chunks
    GateBuf<64> G[2];                              // by chunk parity
    float red[kWaves][64];                         // q^ . X partial sums per wave
};
static_assert(sizeof(WalkSmem) <= 160 * 1024, "LDS budget");

struct WalkArgs {
    const uint16_t* q;    // [S, T, DQK] rows
    const uint16_t* k;
    const uint16_t* v;
    const uint16_t* dh;   // [S, T, DV] rows
    const float* ipre;
    const float* fpre;
    const float* C0;      // entry state of segment 0 (NULL: zero state, m = m0 or 0)
    const float* n0;
    const float* m0;
    const float* seg;     // segment slots of the local pass and the combine (G > 1)
    float* out;           // S (NC - 1) chunk slots: n and m entering chunk c >= 1 in slot c - 1
    float* X;             // kNTile x [S, T, DQK]: X^T partial sums over each tile's columns
    float* part;          // [S, T, part_stride]: q^ . X partial sum of tile j at offset j
    int part_stride;
    int S;
    int T;
    int G;                // segments per sequence
    int R;                // local sub-segments per segment; segment g >= 1 enters from slot g R - 1
    int NS;               // segment slots per sequence, (G - 1) R
    int seg_chunks;       // chunks per segment (the last may be shorter)
    uint32_t nh_magic;    // as in ChunkKernelArgs
    int64_t sk[2], sv[2];
    uint32_t rk, rv;
};

// the chunk's K rows, both d blocks: two 16-byte pieces per thread and block
constexpr int kWalkKP = 64 * (Cfg<64>::DB / 8) / kThreads;
__device__ __forceinline__ void walk_load_k(u32x4_t (&r)[Cfg<64>::NDB][kWalkKP], const SeqRsrc& R, int t0, int tid,
                                            uint32_t rk) {
    constexpr int PR = Cfg<64>::DB / 8;
#pragma unroll
    for (int p = 0; p < Cfg<64>::NDB; ++p)
#pragma unroll
        for (int i = 0; i < kWalkKP; ++i) {
            const int item = tid + i * kThreads;
            r[p][i] = bload128(R.k, static_cast<uint32_t>(t0 + item / PR) * rk + 16 * (item % PR), p * Cfg<64>::DB * 2);
        }
}
__device__ __forceinline__ void walk_store_k(WalkSmem& S, const u32x4_t (&r)[Cfg<64>::NDB][kWalkKP], int tid) {
    constexpr int PR = Cfg<64>::DB / 8;
#pragma unroll
    for (int p = 0; p < Cfg<64>::NDB; ++p)
#pragma unroll
        for (int i = 0; i < kWalkKP; ++i) {
            const int item = tid + i * kThreads;
            const int off = (item / PR) * Cfg<64>::QP + 8 * (item % PR);
            MLSTM_CHECK(off + 8 <= 64 * Cfg<64>::QP, kDbgChunkBwd);
            *reinterpret_cast<u32x4_t*>(&S.K[p][off]) = r[p][i];
        }
}
// the chunk's dH rows, this tile's 128 columns: two 16-byte pieces per thread
__device__ __forceinline__ void walk_load_dh(u32x4_t (&r)[2], __amdgpu_buffer_rsrc_t rdh, int t0, int v0, int tid) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int item = tid + i * kThreads;
        r[i] = bload128(rdh, static_cast<uint32_t>((t0 + item / 16) * kDV + v0 + 8 * (item % 16)) * 2u, 0);
    }
}
__device__ __forceinline__ void walk_store_dh(WalkSmem& S, const u32x4_t (&r)[2], int tid) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int item = tid + i * kThreads;
        *reinterpret_cast<u32x4_t*>(&S.dH[(item / 16) * kWalkHP + 8 * (item % 16)]) = r[i];
    }
}
// (w V)^T from the packed V^T as a bf16 pair: hi = bf16(w v), lo = bf16(w v - hi)
__device__ __forceinline__ void vt_store_hilo(WalkSmem& S, const VtPacked<64>& pv, const float* wC, int wave, int lane) {
    constexpr int TP = Cfg<64>::TP, NA = 64 / 16;
    const int l16 = lane & 15, g16 = lane >> 4;
#pragma unroll
    for (int i = 0; i < VRegs<64>::N * VRegs<64>::PARTS; ++i) {
        const int pc = wave + kWaves * i, a = pc % NA, b = pc / NA;
        const int tau = 16 * a + 4 * g16;
        const f32x4_t w = *reinterpret_cast<const f32x4_t*>(&wC[tau]);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const u32x2_t x = pv[2 * i + h];
            const float f0 = lo_f32(x[0]) * w[0], f1 = hi_f32(x[0]) * w[1];
            const float f2 = lo_f32(x[1]) * w[2], f3 = hi_f32(x[1]) * w[3];
            u32x2_t oh, ol;
            oh[0] = pack_bf16x2(f0, f1);
            oh[1] = pack_bf16x2(f2, f3);
            ol[0] = pack_bf16x2(f0 - lo_f32(oh[0]), f1 - hi_f32(oh[0]));
            ol[1] = pack_bf16x2(f2 - lo_f32(oh[1]), f3 - hi_f32(oh[1]));
            const int row = 32 * b + 16 * h + l16;
            MLSTM_CHECK(row < kDVT && tau + 4 <= TP, kDbgChunkBwd);
            *reinterpret_cast<u32x2_t*>(&S.Vw[0][row * TP + tau]) = oh;
            *reinterpret_cast<u32x2_t*>(&S.Vw[1][row * TP + tau]) = ol;
        }
    }
}

__global__ void __launch_bounds__(kThreads, 1) bwd_walk_kernel(WalkArgs A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    WalkSmem& S = *reinterpret_cast<WalkSmem*>(smem_raw);
    constexpr int L = 64;
    using CF = Cfg<64>;
    constexpr int QP = CF::QP, TP = CF::TP, DB = CF::DB, NDB = CF::NDB;
    constexpr int NKS = L / 32;
    static_assert(DB / 16 == kWaves, "one n-update tile per wave and d block");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, l16 = lane & 15;
    const bool gate_wave = (wave == kGateWave);

    const int wi = work_index();
    const int tile = wi % kNTile;
    const int sg = wi / kNTile;
    const int g = sg % A.G;
    const int s = sg / A.G;
    const int v0 = tile * kDVT;
    const int nc_total = (A.T + L - 1) / L;
    const int c_begin = g * A.seg_chunks;
    const int c_end = min(nc_total, c_begin + A.seg_chunks);
    MLSTM_CHECK(s < A.S, kDbgChunkBwd);
    const int64_t st = static_cast<int64_t>(s) * A.T;

    SeqRsrc P;
    P.k = make_rsrc(seq_rows(A.k, s, A.nh_magic, A.sk), seq_span(A.T, A.rk, kDQK));
    P.v = make_rsrc(seq_rows(A.v, s, A.nh_magic, A.sv), seq_span(A.T, A.rv, kDV));
    P.ig = make_rsrc(A.ipre + st, static_cast<uint32_t>(A.T) * 4);
    P.fg = make_rsrc(A.fpre + st, static_cast<uint32_t>(A.T) * 4);
    const __amdgpu_buffer_rsrc_t rdh = make_rsrc(A.dh + st * kDV, static_cast<uint32_t>(A.T) * kDV * 2);
    float* Xt = A.X + static_cast<int64_t>(tile) * A.S * A.T * kDQK;

    // entry state into the C^T tiles: Ct[dt][pp][e][j] = C[dw(dt) + l16][v0 + 32 pp + 8 g16 + 4 e + j]
    auto dw = [&](int dt) { return 32 * wave + 16 * dt; };
    f32x4_t Ct[2][4][2];
    const float* nin;
    float m_prev;
    if (g == 0) {
        const float* C0 = A.C0 ? A.C0 + static_cast<int64_t>(s) * kDQK * kDV : nullptr;
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
            for (int pp = 0; pp < 4; ++pp)
#pragma unroll
                for (int e = 0; e < 2; ++e)
                    Ct[dt][pp][e] = C0 ? *reinterpret_cast<const f32x4_t*>(
                                             C0 + static_cast<int64_t>(dw(dt) + l16) * kDV + v0 + 32 * pp + 8 * g16 + 4 * e)
                                       : f32x4_t{};
        nin = A.n0 ? A.n0 + static_cast<int64_t>(s) * kDQK : nullptr;
        m_prev = A.m0 ? A.m0[s] : 0.0f;
    } else {
        MLSTM_CHECK(g * A.R - 1 >= 0 && g * A.R - 1 < A.NS, kDbgChunkBwd);
        const float* slot = A.seg + (static_cast<int64_t>(s) * A.NS + g * A.R - 1) * kSlotFloats;
        // the slot holds four rows interleaved: element (d, v) at slot_c4(d / 4, v) + d % 4
#pragma unroll
        for (int dt = 0; dt < 2; ++dt) {
            const int d = dw(dt) + l16;
#pragma unroll
            for (int pp = 0; pp < 4; ++pp)
#pragma unroll
                for (int e = 0; e < 2; ++e)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        Ct[dt][pp][e][j] = slot[slot_c4(d / 4, v0 + 32 * pp + 8 * g16 + 4 * e + j) + d % 4];
        }
        nin = slot + kDQK * kDV;
        m_prev = slot[kDQK * kDV + kDQK + 2];
    }
    if (tid < kDQK) S.n[0][tid] = nin ? nin[tid] : 0.0f;
    float s_off = 0.0f;   // C = C_acc e^{s_off}
    float g_m = m_prev, g_s = 0.0f;
    float gi[2] = {0.f, 0.f}, gf[2] = {0.f, 0.f};

    u32x4_t rk[NDB][kWalkKP];
    u32x4_t rdhv[2];
    VRegs<64> rv;
    VtPacked<64> pv;
    if (c_begin < c_end) {
        const int t0 = c_begin * L;
        walk_load_k(rk, P, t0, tid, A.rk);
        load_v_tr<64>(rv, P, t0, v0, wave, lane, 0, A.rv);
        walk_load_dh(rdhv, rdh, t0, v0, tid);
        if (gate_wave) {
            load_gates<64>(gi, gf, P, t0, lane);
            gate_phase<64>(S.G[c_begin & 1], gi, gf, g_m, g_s, lane, A.T - t0);
        }
    }

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * L;
        const int cur = (c - c_begin) & 1;
        const int par = c & 1;
        const GateBuf<64>& Gc = S.G[par];
        __syncthreads();   // the previous chunk is done; this chunk's gates and n are visible
        if (c > c_begin && tid < L && t0 - L + tid < A.T) {
            // the previous chunk's q^ . X share of this tile
            float qx = 0.0f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) qx += S.red[w][tid];
            A.part[(st + t0 - L + tid) * A.part_stride + tile] = qx;
        }
        walk_store_k(S, rk, tid);
        walk_store_dh(S, rdhv, tid);
        vt_transpose<64>(pv, rv, lane, 0);
        vt_store_hilo(S, pv, Gc.wC, wave, lane);
        if (c + 1 < c_end) {
            walk_load_k(rk, P, t0 + L, tid, A.rk);
            load_v_tr<64>(rv, P, t0 + L, v0, wave, lane, 0, A.rv);
            walk_load_dh(rdhv, rdh, t0 + L, v0, tid);
            if (gate_wave) load_gates<64>(gi, gf, P, t0 + L, lane);
        }
        if (c > 0 && tile == 0) {
            // n and m entering chunk c
            MLSTM_CHECK(c - 1 < nc_total - 1, kDbgChunkBwd);
            float* slot = A.out + (static_cast<int64_t>(s) * (nc_total - 1) + c - 1) * kSlotFloats;
            if (tid < kDQK) slot[kDQK * kDV + tid] = S.n[cur][tid];
            if (tid == 0) slot[kDQK * kDV + kDQK + 2] = m_prev;
        }
        __syncthreads();   // the chunk's K rows, dH rows and weighted V^T are visible
        // gates of the next chunk, one chunk ahead
        if (gate_wave && c + 1 < c_end) gate_phase<64>(S.G[par ^ 1], gi, gf, g_m, g_s, lane, A.T - (t0 + L));

        // X^T [d][tau] = sum_v C[d][v] dH[tau][v] over this tile's columns, C as a bf16 pair hi + lo
        {
            // the q rows of q^ . X, requested before the products so that their latency is covered
            u32x2_t qv[2][4];
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int tb = 0; tb < 4; ++tb) {
                    const int tau = 16 * tb + l16;
                    qv[dt][tb] = (t0 + tau < A.T)
                                     ? *reinterpret_cast<const u32x2_t*>(A.q + (st + t0 + tau) * kDQK + dw(dt) + 4 * g16)
                                     : u32x2_t{0u, 0u};
                }
            f32x4_t X[2][4];
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int tb = 0; tb < 4; ++tb) X[dt][tb] = f32x4_t{};
#pragma unroll
            for (int pp = 0; pp < 4; ++pp) {
                u32x4_t b[4];
#pragma unroll
                for (int tb = 0; tb < 4; ++tb)
                    b[tb] = *reinterpret_cast<const u32x4_t*>(&S.dH[(16 * tb + l16) * kWalkHP + 32 * pp + 8 * g16]);
#pragma unroll
                for (int dt = 0; dt < 2; ++dt) {
                    const f32x4_t& c0 = Ct[dt][pp][0];
                    const f32x4_t& c1 = Ct[dt][pp][1];
                    u32x4_t ah, al;
                    ah[0] = pack_bf16x2(c0[0], c0[1]);
                    ah[1] = pack_bf16x2(c0[2], c0[3]);
                    ah[2] = pack_bf16x2(c1[0], c1[1]);
                    ah[3] = pack_bf16x2(c1[2], c1[3]);
                    al[0] = pack_bf16x2(c0[0] - lo_f32(ah[0]), c0[1] - hi_f32(ah[0]));
                    al[1] = pack_bf16x2(c0[2] - lo_f32(ah[1]), c0[3] - hi_f32(ah[1]));
                    al[2] = pack_bf16x2(c1[0] - lo_f32(ah[2]), c1[1] - hi_f32(ah[2]));
                    al[3] = pack_bf16x2(c1[2] - lo_f32(ah[3]), c1[3] - hi_f32(ah[3]));
#pragma unroll
                    for (int tb = 0; tb < 4; ++tb) {
                        X[dt][tb] = mfma16(ah, b[tb], X[dt][tb]);
                        X[dt][tb] = mfma16(al, b[tb], X[dt][tb]);
                    }
                }
            }
            // C = C_acc e^{s}; lane (tau = 16 tb + l16, g16) holds X^T[dw(dt) + 4 g16 + 0..3][tau]
            const float esc = expf(s_off);
            float qx[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int dt = 0; dt < 2; ++dt) {
                const int d = dw(dt) + 4 * g16;
#pragma unroll
                for (int tb = 0; tb < 4; ++tb) {
                    const int tau = 16 * tb + l16;
                    if (t0 + tau < A.T) {
                        const f32x4_t x = X[dt][tb] * esc;
                        *reinterpret_cast<f32x4_t*>(Xt + (st + t0 + tau) * kDQK + d) = x;
                        const u32x2_t q = qv[dt][tb];
                        qx[tb] += lo_f32(q[0]) * x[0] + hi_f32(q[0]) * x[1] + lo_f32(q[1]) * x[2] + hi_f32(q[1]) * x[3];
                    }
                }
            }
#pragma unroll
            for (int tb = 0; tb < 4; ++tb) {
                const float v = sum_rows4(qx[tb]);
                if (g16 == 0) S.red[wave][16 * tb + l16] = v * kQScale;
            }
        }

        const float decay_n = Gc.scal[0];
        const float m_next = Gc.scal[1];
        const float s_new = Gc.scal[2];
        const float c_scale = Gc.scal[3];   // != 1: apply this chunk's decay to C_acc eagerly
        if (c_scale != 1.0f) {
#pragma unroll
            for (int dt = 0; dt < 2; ++dt)
#pragma unroll
                for (int pp = 0; pp < 4; ++pp)
#pragma unroll
                    for (int e = 0; e < 2; ++e) Ct[dt][pp][e] *= c_scale;
        }
        const int tr_row = (l16 >> 2) + 8 * g16;
        const int tr_col = 4 * (l16 & 3);
        // C^T += (w e^{-s} V)^T K (hi, then lo): A = the weighted V^T rows in the pair order (row l16 of
        // tile (pp, e) is v = 32 pp + 8 (l16 / 4) + 4 e + l16 % 4), B = K read transposed (this wave's d)
        {
            const uint16_t* Ks = S.K[wave / 4];
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                u32x4_t kt[2];
#pragma unroll
                for (int dt = 0; dt < 2; ++dt) {
                    const uint16_t* kb = &Ks[(32 * ks + tr_row) * QP + 32 * (wave % 4) + 16 * dt + tr_col];
                    kt[dt] = cat(tr_read(kb), tr_read(kb + 4 * QP));
                }
#pragma unroll
                for (int pp = 0; pp < 4; ++pp)
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int off = (32 * pp + 8 * (l16 >> 2) + 4 * e + (l16 & 3)) * TP + 32 * ks + 8 * g16;
                        const u32x4_t vh = *reinterpret_cast<const u32x4_t*>(&S.Vw[0][off]);
                        const u32x4_t vl = *reinterpret_cast<const u32x4_t*>(&S.Vw[1][off]);
#pragma unroll
                        for (int dt = 0; dt < 2; ++dt) {
                            Ct[dt][pp][e] = mfma16(vh, kt[dt], Ct[dt][pp][e]);
                            Ct[dt][pp][e] = mfma16(vl, kt[dt], Ct[dt][pp][e]);
                        }
                    }
            }
        }
        // n_p = decay n_p + K_p^T w over this wave's 16 columns of each block: A = w as bf16 hi / lo
        // rows, B = K read transposed
        const float* n_old = S.n[cur];
        float* n_new = S.n[cur ^ 1];
#pragma unroll
        for (int p = 0; p < NDB; ++p) {
            const uint16_t* Ks = S.K[p];
            f32x4_t nacc = f32x4_t{};
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) {
                const u32x4_t wa = (l16 < 2) ? *reinterpret_cast<const u32x4_t*>(&Gc.wb[l16 & 1][32 * ks + 8 * g16])
                                             : u32x4_t{0u, 0u, 0u, 0u};
                const uint16_t* kb = &Ks[(32 * ks + tr_row) * QP + 16 * wave + tr_col];
                nacc = mfma16(wa, cat(tr_read(kb), tr_read(kb + 4 * QP)), nacc);
            }
            if (g16 == 0) {
                const int d = p * DB + 16 * wave + l16;
                n_new[d] = decay_n * n_old[d] + nacc[0] + nacc[1];
            }
        }
        s_off = s_new;
        m_prev = m_next;
    }
    __syncthreads();
    if (c_begin < c_end && tid < L) {
        const int t0 = (c_end - 1) * L;   // the last chunk's q^ . X share
        if (t0 + tid < A.T) {
            float qx = 0.0f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) qx += S.red[w][tid];
            A.part[(st + t0 + tid) * A.part_stride + tile] = qx;
        }
    }
}

hipError_t launch_walk(const WalkArgs& a, hipStream_t stream) {
    const size_t lds = sizeof(WalkSmem);
    static std::atomic<uint64_t> raised{0};
    hipError_t e = raise_dynamic_lds(reinterpret_cast<const void*>(bwd_walk_kernel), lds, raised);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bwd_walk_kernel, dim3(static_cast<unsigned>(a.S * a.G * kNTile)), dim3(kThreads), lds, stream,
                       a);
    return hipGetLastError();
}

// The walk after the prefill's segment schedule (local pass in the bf16 hi + lo form, combine), which
// gives the entry states of the segments; q, k, v and dh are contiguous [S, T, D] rows.
size_t bwd_walk_workspace_bytes(int64_t S, int T) {
    return chunk_mfma_workspace_bytes(static_cast<int>(S), 1, T, kDQK, kDV, kBL);
}

hipError_t launch_bwd_walk(const ChunkArgs& a, const void* dh, float* slots, float* seg, float* X, float* part,
                           hipStream_t stream) {
    if (a.T == 0) return hipSuccess;
    const SegmentShape sh = segment_shape(a.B, a.NH, a.T, kBL, seg != nullptr);
    hipError_t e = launch_segment_states(a, kBL, sh, seg, true, stream);
    if (e != hipSuccess) return e;
    WalkArgs w{};
    w.q = static_cast<const uint16_t*>(a.q);
    w.k = static_cast<const uint16_t*>(a.k);
    w.v = static_cast<const uint16_t*>(a.v);
    w.dh = static_cast<const uint16_t*>(dh);
    w.nh_magic = 0;
    w.sk[0] = 0;
    w.sk[1] = static_cast<int64_t>(a.T) * kDQK;
    w.sv[0] = 0;
    w.sv[1] = static_cast<int64_t>(a.T) * kDV;
    w.rk = kDQK * 2;
    w.rv = kDV * 2;
    w.ipre = a.ipre;
    w.fpre = a.fpre;
    w.C0 = a.C0;
    w.n0 = a.n0;
    w.m0 = a.m0;
    w.seg = seg;
    w.out = slots;
    w.X = X;
    w.part = part;
    w.part_stride = kPartF;
    w.S = a.B * a.NH;
    w.T = a.T;
    w.G = sh.G;
    w.R = sh.R;
    w.NS = (sh.G - 1) * sh.R;
    w.seg_chunks = sh.seg_chunks;
    return launch_walk(w, stream);
}

// ---- X: the sum of the walk's tile partials, into dq ---------------------------------------------
__global__ void __launch_bounds__(256) bwd_xsum_kernel(const float* __restrict__ X, float* __restrict__ dq, int64_t n4) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n4) return;
    const f32x4_t* x = reinterpret_cast<const f32x4_t*>(X);
    reinterpret_cast<f32x4_t*>(dq)[i] = (x[i] + x[n4 + i]) + (x[2 * n4 + i] + x[3 * n4 + i]);
}

// ---- intra pass --------------------------------------------------------------------------------
struct IntraSmem {
    uint16_t Q[kBL * kQP];
    uint16_t K[kBL * kQP];
    uint16_t dH[kBL * kWP];    // one 128-column piece of dH
    uint16_t dHg[kBL * kWP];   // the same piece scaled by g / den / sqrt(DQK)
    uint16_t V[kBL * kWP];     // the same piece of V
    uint16_t P[2][kBL * kPP];  // P [tau][sigma] as bf16 hi and lo
    uint16_t Sn[kBL * kPP];    // St / den [tau][sigma]
    float n[kDQK];
    float x[kBL];
    float M[kBL];
    float gd[kBL];
    float gw[kBL];
    int R[kBL];
    float red[4][kBL];
};
static_assert(sizeof(IntraSmem) <= 160 * 1024, "LDS budget");

// One workgroup per chunk (4 waves).  Wave w owns the tau block w of every [sigma][tau] tile.
__global__ void __launch_bounds__(kBT) bwd_intra_kernel(BwdParams A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    IntraSmem& S = *reinterpret_cast<IntraSmem*>(smem_raw);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, l16 = lane & 15;
    const int c = blockIdx.x % A.NC, s = blockIdx.x / A.NC;
    const int T = A.T, t0 = c * kBL;
    const int64_t st = static_cast<int64_t>(s) * T;
    const auto rq = make_rsrc(A.q + st * kDQK, static_cast<uint32_t>(T) * kDQK * 2);
    const auto rk = make_rsrc(A.k + st * kDQK, static_cast<uint32_t>(T) * kDQK * 2);
    const auto rv = make_rsrc(A.v + st * kDV, static_cast<uint32_t>(T) * kDV * 2);
    const auto rdh = make_rsrc(A.dh + st * kDV, static_cast<uint32_t>(T) * kDV * 2);
    float* lz = lz_of(A, s, c);   // chunk >= 1: the slot holding the entry state (n, m read first)

    float m_prev;
    if (c) {
        m_prev = lz[kCV + kDQK + 2];
        S.n[tid] = lz[kCV + tid];
    } else {
        m_prev = A.m0 ? A.m0[s] : 0.0f;
        S.n[tid] = A.n0 ? A.n0[static_cast<int64_t>(s) * kDQK + tid] : 0.0f;
    }
    stage_rows<kDQK>(S.Q, kQP, rq, kDQK, t0, 0, tid);
    stage_rows<kDQK>(S.K, kQP, rk, kDQK, t0, 0, tid);
    if (wave == 0) {
        BGate G;
        float decay;
        bwd_gates(make_rsrc(A.ipre + st, static_cast<uint32_t>(T) * 4), make_rsrc(A.fpre + st, static_cast<uint32_t>(T) * 4),
                  T, t0, m_prev, lane, G, decay);
        S.x[lane] = G.x;
        S.M[lane] = G.M;
        S.R[lane] = G.R;
        S.gw[lane] = G.g;   // g for now; g w below
        S.gd[lane] = G.fl;  // floor for now; g / den below
        if (t0 + lane < T) A.tok[(st + t0 + lane) * kTokF] = G.wk;
        if (lane == 0) A.chunk[static_cast<int64_t>(s) * A.NC + c] = decay;
    }
    __syncthreads();

    // S^T tiles of this wave: columns tau = 16 wave + l16, rows sigma = 16 j + 4 g16 + 0..3 (j <= wave)
    const int tau = 16 * wave + l16;
    const bool valid = t0 + tau < T;
    f32x4_t Sa[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) Sa[j] = f32x4_t{};
#pragma unroll
    for (int j = 0; j < 4; ++j)
        if (j <= wave)
#pragma unroll
            for (int ks = 0; ks < kDQK / 32; ++ks)
                Sa[j] = mfma16(row_op(S.K, kQP, 16 * j, 32 * ks, lane), row_op(S.Q, kQP, 16 * wave, 32 * ks, lane), Sa[j]);
    const float Mt = S.M[tau];
    const int Rt = S.R[tau];
    const float gt = S.gw[tau];
    const float flt = S.gd[tau];
    float Et[4][4];
    float rsum = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int sg = 16 * j + 4 * g16 + r;
            const float xs = S.x[sg];
            const float e = (sg <= tau && sg >= Rt && xs != -INFINITY) ? fexp(xs - Mt) : 0.0f;
            Et[j][r] = e;
            Sa[j][r] = Sa[j][r] * kQScale * e;
            rsum += Sa[j][r];
        }
    rsum = sum_rows4(rsum);
    float qn = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const u32x4_t qv = lds16(&S.Q[tau * kQP + 64 * g16 + 8 * i]);
#pragma unroll
        for (int e = 0; e < 8; ++e) qn += bf_at(qv, e) * S.n[64 * g16 + 8 * i + e];
    }
    qn = sum_rows4(qn) * kQScale;
    const float Dt = gt * qn + rsum;
    const float den = fmaxf(fabsf(Dt), flt);
    const bool act = fabsf(Dt) > flt;
    const float rden = 1.0f / den;
    const float gd = valid ? gt * rden : 0.0f;
    __syncthreads();   // floor and g are read by every wave
    if (g16 == 0) S.gd[tau] = gd;
    // St / den as bf16 [tau][sigma] (zero above the diagonal)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t p0 = pack_bf16x2(Sa[j][0] * rden, Sa[j][1] * rden);
        const uint32_t p1 = pack_bf16x2(Sa[j][2] * rden, Sa[j][3] * rden);
        *reinterpret_cast<u32x2_t*>(&S.Sn[tau * kPP + 16 * j + 4 * g16]) = u32x2_t{p0, p1};
    }

    // dv pieces of 128 columns: Ap = (V dH^T)^T accumulates;
    //   dv_i^T [v][sigma] = sum_tau dH^T[v][tau] (St / den)[tau][sigma]
    //   L_c^T  [v][d]     = sum_tau (g / den dH)^T[v][tau] Q^[tau][d]
    f32x4_t Ap[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) Ap[j] = f32x4_t{};
    for (int pc = 0; pc < kDV / 128; ++pc) {
        __syncthreads();   // the previous piece is consumed; Sn and gd are visible
        {
            constexpr int N = kBL * 16 / kBT;
            u32x4_t tmp[N];
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int e = tid + kBT * i, row = e / 16, p8 = e % 16;
                tmp[i] = bload128(rdh, static_cast<uint32_t>((t0 + row) * kDV + 128 * pc + 8 * p8) * 2u, 0);
            }
#pragma unroll
            for (int i = 0; i < N; ++i) {
                const int e = tid + kBT * i, row = e / 16, p8 = e % 16;
                *reinterpret_cast<u32x4_t*>(&S.dH[row * kWP + 8 * p8]) = tmp[i];
                const float sc = S.gd[row] * kQScale;
                u32x4_t o;
#pragma unroll
                for (int w = 0; w < 4; ++w) o[w] = pack_bf16x2(lo_f32(tmp[i][w]) * sc, hi_f32(tmp[i][w]) * sc);
                *reinterpret_cast<u32x4_t*>(&S.dHg[row * kWP + 8 * p8]) = o;
            }
        }
        stage_rows<128>(S.V, kWP, rv, kDV, t0, 128 * pc, tid);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (j <= wave)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    Ap[j] = mfma16(row_op(S.V, kWP, 16 * j, 32 * ks, lane), row_op(S.dH, kWP, 16 * wave, 32 * ks, lane), Ap[j]);
#pragma unroll
        for (int vb = 0; vb < 2; ++vb) {
            const int vloc = 16 * (2 * wave + vb);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f32x4_t acc = f32x4_t{};
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
                    if (32 * ks + 31 >= 16 * j)
                        acc = mfma16(tr_op(S.dH, kWP, 32 * ks, vloc, lane), tr_op(S.Sn, kPP, 32 * ks, 16 * j, lane), acc);
                const int sg = 16 * j + l16;
                if (t0 + sg < T)
                    *reinterpret_cast<f32x4_t*>(&A.dv[(st + t0 + sg) * kDV + 128 * pc + vloc + 4 * g16]) = acc;
            }
        }
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            f32x4_t La[2][8];
#pragma unroll
            for (int vb = 0; vb < 2; ++vb)
#pragma unroll
                for (int db = 0; db < 8; ++db) La[vb][db] = f32x4_t{};
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                u32x4_t a[2];
#pragma unroll
                for (int vb = 0; vb < 2; ++vb) a[vb] = tr_op(S.dHg, kWP, 32 * ks, 16 * (2 * wave + vb), lane);
#pragma unroll
                for (int db = 0; db < 8; ++db) {
                    const u32x4_t b = tr_op(S.Q, kQP, 32 * ks, 16 * (8 * half + db), lane);
#pragma unroll
                    for (int vb = 0; vb < 2; ++vb) La[vb][db] = mfma16(a[vb], b, La[vb][db]);
                }
            }
#pragma unroll
            for (int vb = 0; vb < 2; ++vb)
#pragma unroll
                for (int db = 0; db < 8; ++db)
                    *reinterpret_cast<f32x4_t*>(&lz[static_cast<int64_t>(16 * (8 * half + db) + l16) * kDV + 128 * pc +
                                                    16 * (2 * wave + vb) + 4 * g16]) = La[vb][db];
        }
    }
    // dh_t . N_t from its two parts: the entry state's g q^_t . (dH C^T)_t (the dhc pass's partial
    // sums) and the intra sum_sigma St_t,sigma (dh_t . v_sigma); then w_t
    float dhn = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) dhn += Sa[j][r] * Ap[j][r];
    dhn = sum_rows4(dhn);
    float qx = 0.0f;
    if (valid) {
        const float* pp = &A.part[(st + t0 + tau) * kPartF];
        qx = (pp[0] + pp[1]) + (pp[2] + pp[3]);
    }
    dhn += gt * qx;
    const float wt = (act && valid) ? -(dhn * rden) * (Dt > 0.0f ? 1.0f : -1.0f) * rden : 0.0f;
    const float gwt = gt * wt;
    if (g16 == 0) S.gw[tau] = gwt;
    // P^T [sigma][tau] = E o (A'^T / den + w), stored as P [tau][sigma] in bf16 hi + lo: where the
    // numerator and denominator terms of a row nearly cancel, P's own rounding would show
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        float pv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) pv[r] = Et[j][r] * (Ap[j][r] * rden + wt);
        const uint32_t h01 = pack_bf16x2(pv[0], pv[1]), h23 = pack_bf16x2(pv[2], pv[3]);
        *reinterpret_cast<u32x2_t*>(&S.P[0][tau * kPP + 16 * j + 4 * g16]) = u32x2_t{h01, h23};
        *reinterpret_cast<u32x2_t*>(&S.P[1][tau * kPP + 16 * j + 4 * g16]) =
            u32x2_t{pack_bf16x2(pv[0] - lo_f32(h01), pv[1] - hi_f32(h01)),
                    pack_bf16x2(pv[2] - lo_f32(h23), pv[3] - hi_f32(h23))};
    }
    __syncthreads();
    // dq^T [d][tau] = (g / den X + sum_sigma K^T[d][sigma] P^T[sigma][tau] + g w n) / sqrt(DQK), X (in
    // dq) the sum of the walk's four tile partials; r_t = q_t . dq_t
    float rpart[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < 4; ++db) {
        const int d0 = 16 * (4 * wave + db);
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
            f32x4_t acc = f32x4_t{};
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
                if (32 * ks <= 16 * tb + 15) {
                    const u32x4_t a = tr_op(S.K, kQP, 32 * ks, d0, lane);
                    acc = mfma16(a, row_op(S.P[0], kPP, 16 * tb, 32 * ks, lane), acc);
                    acc = mfma16(a, row_op(S.P[1], kPP, 16 * tb, 32 * ks, lane), acc);
                }
            const int tt = 16 * tb + l16;
            if (t0 + tt < T) {
                const float gw_t = S.gw[tt], gd_t = S.gd[tt];
                const int d = d0 + 4 * g16;
                float* dqp = &A.dq[(st + t0 + tt) * kDQK + d];
                const f32x4_t x = *reinterpret_cast<const f32x4_t*>(dqp);
                f32x4_t o;
#pragma unroll
                for (int r = 0; r < 4; ++r) o[r] = (gd_t * x[r] + acc[r] + gw_t * S.n[d + r]) * kQScale;
                *reinterpret_cast<f32x4_t*>(dqp) = o;
                const u32x2_t qv = lds_u32x2(&S.Q[tt * kQP + d]);
                rpart[tb] += lo_f32(qv[0]) * o[0] + hi_f32(qv[0]) * o[1] + lo_f32(qv[1]) * o[2] + hi_f32(qv[1]) * o[3];
            }
        }
    }
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) {
        const float r = sum_rows4(rpart[tb]);
        if (g16 == 0) S.red[wave][16 * tb + l16] = r;
    }
    // dk_i^T [d][sigma] = sum_tau Q^T[d][tau] P[tau][sigma] / sqrt(DQK)
#pragma unroll
    for (int db = 0; db < 4; ++db) {
        const int d0 = 16 * (4 * wave + db);
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            f32x4_t acc = f32x4_t{};
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
                if (32 * ks + 31 >= 16 * sb) {
                    const u32x4_t a = tr_op(S.Q, kQP, 32 * ks, d0, lane);
                    acc = mfma16(a, tr_op(S.P[0], kPP, 32 * ks, 16 * sb, lane), acc);
                    acc = mfma16(a, tr_op(S.P[1], kPP, 32 * ks, 16 * sb, lane), acc);
                }
            const int sg = 16 * sb + l16;
            if (t0 + sg < T) {
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[r] *= kQScale;
                *reinterpret_cast<f32x4_t*>(&A.dk[(st + t0 + sg) * kDQK + d0 + 4 * g16]) = acc;
            }
        }
    }
    // z_c = Q^T (g o w) / sqrt(DQK) into the chunk's L slot (its n was read at the start)
    {
        float z = 0.0f;
        for (int t = 0; t < kBL; ++t) z += bf16_to_f32(S.Q[t * kQP + tid]) * S.gw[t];
        lz[kCV + tid] = z * kQScale;
    }
    __syncthreads();
    if (tid < kBL && t0 + tid < T) {
        float* pp = &A.part[(st + t0 + tid) * kPartF];
        pp[0] = S.red[0][tid] + S.red[1][tid] + S.red[2][tid] + S.red[3][tid];
        pp[1] = 0.0f;
        pp[2] = 0.0f;
        pp[3] = 0.0f;
    }
}

// ---- reverse scan of the state gradient --------------------------------------------------------
__global__ void __launch_bounds__(256) bwd_scan_kernel(BwdParams A) {
    const int s = blockIdx.y;
    const int e4 = blockIdx.x * 256 + threadIdx.x;
    const bool ok = e4 < kScanE4;
    const bool isC = e4 < kCV / 4;
    const int NC = A.NC;
    f32x4_t G = f32x4_t{};
    constexpr int kBatch = 8;
    for (int c1 = NC - 1; c1 >= 0; c1 -= kBatch) {
        const int nb = min(kBatch, c1 + 1);
        f32x4_t Lv[kBatch];
        float dec[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (u < nb) {
                const int c = c1 - u;
                dec[u] = A.chunk[static_cast<int64_t>(s) * NC + c];
                if (ok) Lv[u] = reinterpret_cast<const f32x4_t*>(lz_of(A, s, c))[e4];
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (u < nb) {
                const int c = c1 - u;
                if (ok && c < NC - 1) {
                    if (isC) {
                        // one bf16 rounding, like the other operands of the bf16 products: the
                        // inter terms of dk and dv sum it against v and k (a hi + lo pair measured
                        // 1.5 x smaller row errors, at twice the traffic of this pass and the next)
                        uint16_t* hb = hl_of(A, s, c) + 4 * static_cast<int64_t>(e4);
                        *reinterpret_cast<u32x2_t*>(hb) = u32x2_t{pack_bf16x2(G[0], G[1]), pack_bf16x2(G[2], G[3])};
                    } else {
                        reinterpret_cast<f32x4_t*>(A.gamn + (static_cast<int64_t>(s) * NC + c) * kDQK)[e4 - kCV / 4] = G;
                    }
                }
                if (ok) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) G[r] = dec[u] * G[r] + Lv[u][r];
                }
            }
        }
    }
    // Gam_{-1}, gam_{-1}: the gradients of C0 and n0, and this block's share of dm0
    if (A.dC0 == nullptr) return;
    float dm = 0.0f;
    if (ok) {
        if (isC) {
            reinterpret_cast<f32x4_t*>(A.dC0 + static_cast<int64_t>(s) * kCV)[e4] = G;
            if (A.C0) {
                const f32x4_t c0 = reinterpret_cast<const f32x4_t*>(A.C0 + static_cast<int64_t>(s) * kCV)[e4];
                dm = G[0] * c0[0] + G[1] * c0[1] + G[2] * c0[2] + G[3] * c0[3];
            }
        } else {
            reinterpret_cast<f32x4_t*>(A.dn0 + static_cast<int64_t>(s) * kDQK)[e4 - kCV / 4] = G;
            if (A.n0) {
                const f32x4_t n0 = reinterpret_cast<const f32x4_t*>(A.n0 + static_cast<int64_t>(s) * kDQK)[e4 - kCV / 4];
                dm = G[0] * n0[0] + G[1] * n0[1] + G[2] * n0[2] + G[3] * n0[3];
            }
        }
    }
    __shared__ float red[4];
    dm = wave_total(dm);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = dm;
    __syncthreads();
    if (threadIdx.x == 0) A.dmp[static_cast<int64_t>(s) * kScanBlocks + blockIdx.x] = red[0] + red[1] + red[2] + red[3];
}

// ---- dk and dv inter terms ---------------------------------------------------------------------
// One workgroup of 8 waves per chunk: dk^T += Gam_c V^T (over v) and dv^T += Gam_c^T K^T (over d),
// each complete inside the workgroup, so Gam_c is read from memory once.  It streams through LDS in
// 16 blocks of 64 rows d x 128 columns v (the next block in registers), while K and V of
// the chunk stay in LDS.  Waves 0-3 form dk: wave m owns the rows d = 64 jd + 16 m + 0..15 of every
// block row jd; waves 4-7 form dv: wave m owns the columns v = 128 jv + 32 m + 0..31 of block column
// jv; both cover the four tau tiles, and each runs 32 MFMAs per block.  The blocks go column by
// column, so a dv wave finishes its columns of jv after four blocks.
constexpr int kIKT = 512;    // threads of the inter pass
struct InterKVSmem {
    uint16_t K[kBL * kQP];     // the chunk's K rows
    uint16_t V[kBL * kHP];     // the chunk's V rows
    uint16_t G[64 * kWP];      // one block of Gam_c
    float wk[kBL];
    float gam[kDQK];
    float red[4][kBL];         // k . dk partials of the dk waves
};
static_assert(sizeof(InterKVSmem) <= 160 * 1024, "LDS budget");

__global__ void __launch_bounds__(kIKT) bwd_interkv_kernel(BwdParams A) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
    InterKVSmem& S = *reinterpret_cast<InterKVSmem*>(smem_raw);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g16 = lane >> 4, l16 = lane & 15;
    const int c = blockIdx.x % A.NC, s = blockIdx.x / A.NC;
    const int T = A.T, t0 = c * kBL;
    const int64_t st = static_cast<int64_t>(s) * T;
    const bool has_g = c < A.NC - 1;   // the last chunk's exit state receives no gradient
    const bool dk_role = wave < 4;
    const int m = wave & 3;

    if (tid < kBL) S.wk[tid] = (t0 + tid < T) ? A.tok[(st + t0 + tid) * kTokF] : 0.0f;
    const uint16_t* gbase = has_g ? hl_of(A, s, c) : nullptr;
    // this thread's two 16-byte pieces of a Gam block (rows e / 16, columns 8 (e % 16) + 0..7)
    u32x4_t gh[2];
    auto gload = [&](int jd, int jv) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int e = tid + kIKT * i;
            const uint16_t* p = gbase + static_cast<int64_t>(64 * jd + (e >> 4)) * kDV + 128 * jv + 8 * (e & 15);
            gh[i] = *reinterpret_cast<const u32x4_t*>(p);
        }
    };
    if (has_g) {
        gload(0, 0);
        const auto rk = make_rsrc(A.k + st * kDQK, static_cast<uint32_t>(T) * kDQK * 2);
        const auto rv = make_rsrc(A.v + st * kDV, static_cast<uint32_t>(T) * kDV * 2);
#pragma unroll
        for (int h = 0; h < 2; ++h) {   // two rounds, so that fewer staging registers are live
            u32x4_t tk[2], tv[4];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int e = tid + kIKT * (2 * h + i), row = e >> 5, pc = e & 31;
                tk[i] = bload128(rk, static_cast<uint32_t>((t0 + row) * kDQK + 8 * pc) * 2u, 0);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = tid + kIKT * (4 * h + i), row = e >> 6, pc = e & 63;
                tv[i] = bload128(rv, static_cast<uint32_t>((t0 + row) * kDV + 8 * pc) * 2u, 0);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int e = tid + kIKT * (2 * h + i), row = e >> 5, pc = e & 31;
                *reinterpret_cast<u32x4_t*>(&S.K[row * kQP + 8 * pc]) = tk[i];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = tid + kIKT * (4 * h + i), row = e >> 6, pc = e & 63;
                *reinterpret_cast<u32x4_t*>(&S.V[row * kHP + 8 * pc]) = tv[i];
            }
        }
        if (tid < kDQK) S.gam[tid] = A.gamn[(static_cast<int64_t>(s) * A.NC + c) * kDQK + tid];
    }

    // dk waves: acc[4 jd + t] (tau tile t); dv waves: acc[4 e + t] (columns 32 m + 16 e of the current
    // block column, tau tile t)
    f32x4_t acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = f32x4_t{};
    if (has_g) {
#pragma unroll 1
        for (int jv = 0; jv < 4; ++jv) {
#pragma unroll
            for (int jd = 0; jd < 4; ++jd) {
                __syncthreads();   // the previous block is consumed (first: K, V, wk, gam staged)
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int e = tid + kIKT * i;
                    *reinterpret_cast<u32x4_t*>(&S.G[(e >> 4) * kWP + 8 * (e & 15)]) = gh[i];
                }
                if (jd < 3) gload(jd + 1, jv);
                else if (jv < 3) gload(0, jv + 1);
                __syncthreads();
                if (dk_role) {
                    // dk^T [d][tau] += sum_v Gam[d][v] V[tau][v]: A = Gam rows, B = V rows
#pragma unroll
                    for (int ks = 0; ks < 4; ++ks) {
                        const u32x4_t ah = row_op(S.G, kWP, 16 * m, 32 * ks, lane);
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            const u32x4_t b = row_op(S.V, kHP, 16 * t, 128 * jv + 32 * ks, lane);
                            acc[4 * jd + t] = mfma16(ah, b, acc[4 * jd + t]);
                        }
                    }
                } else {
                    // dv^T [v][tau] += sum_d Gam[d][v] K[tau][d]: A = Gam read transposed, B = K rows
#pragma unroll
                    for (int ks = 0; ks < 2; ++ks) {
                        u32x4_t ah[2];
#pragma unroll
                        for (int e = 0; e < 2; ++e) ah[e] = tr_op(S.G, kWP, 32 * ks, 32 * m + 16 * e, lane);
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            const u32x4_t b = row_op(S.K, kQP, 16 * t, 64 * jd + 32 * ks, lane);
#pragma unroll
                            for (int e = 0; e < 2; ++e) acc[4 * e + t] = mfma16(ah[e], b, acc[4 * e + t]);
                        }
                    }
                }
            }
            if (!dk_role) {
                // dv of this wave's columns of block column jv: dv += wk (Gam^T K^T)^T
#pragma unroll
                for (int e = 0; e < 2; ++e)
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const int tt = 16 * t + l16;
                        if (t0 + tt < T) {
                            float* dvp = &A.dv[(st + t0 + tt) * kDV + 128 * jv + 32 * m + 16 * e + 4 * g16];
                            f32x4_t o = *reinterpret_cast<const f32x4_t*>(dvp);
                            o += S.wk[tt] * acc[4 * e + t];
                            *reinterpret_cast<f32x4_t*>(dvp) = o;
                        }
                        acc[4 * e + t] = f32x4_t{};
                    }
            }
        }
    } else {
        __syncthreads();   // wk staged
    }
    if (dk_role) {
        // dk += wk (Gam V^T + gam), then this wave's share of k . dk
        float cp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int jd = 0; jd < 4; ++jd) {
            const int d = 64 * jd + 16 * m + 4 * g16;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int tt = 16 * t + l16;
                if (t0 + tt < T) {
                    float* dkp = &A.dk[(st + t0 + tt) * kDQK + d];
                    f32x4_t o = *reinterpret_cast<const f32x4_t*>(dkp);
                    if (has_g) {
                        const float w = S.wk[tt];
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[r] += w * (acc[4 * jd + t][r] + S.gam[d + r]);
                        *reinterpret_cast<f32x4_t*>(dkp) = o;
                    }
                    const u32x2_t kv = *reinterpret_cast<const u32x2_t*>(&A.k[(st + t0 + tt) * kDQK + d]);
                    cp[t] += lo_f32(kv[0]) * o[0] + hi_f32(kv[0]) * o[1] + lo_f32(kv[1]) * o[2] + hi_f32(kv[1]) * o[3];
                }
            }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const float v = sum_rows4(cp[t]);
            if (g16 == 0) S.red[m][16 * t + l16] = v;
        }
    }
    __syncthreads();
    if (tid < kBL && t0 + tid < T) {
        float* pp = &A.part[(st + t0 + tid) * kPartF + 4];
        pp[0] = (S.red[0][tid] + S.red[1][tid]) + (S.red[2][tid] + S.red[3][tid]);
        pp[1] = 0.0f;
        pp[2] = 0.0f;
        pp[3] = 0.0f;
    }
}

// ---- gate gradients ----------------------------------------------------------------------------
constexpr int kGT = 1024;   // threads of the gate pass: one block of kGT tokens per step of its scan
__global__ void __launch_bounds__(kGT) bwd_gate_kernel(BwdParams A) {
    const int s = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int T = A.T;
    const int64_t st = static_cast<int64_t>(s) * T;
    __shared__ float wsum[kGT / 64];
    double carry = 0.0;
    for (int base = ((T + kGT - 1) / kGT - 1) * kGT; base >= 0; base -= kGT) {
        const int t = base + tid;
        float val = 0.0f, ci = 0.0f;
        if (t < T) {
            const float* p = &A.part[(st + t) * kPartF];
            val = (p[0] + p[1]) + (p[2] + p[3]);
            ci = (p[4] + p[5]) + (p[6] + p[7]);
            val -= ci;
        }
        // inclusive prefix over the block, then the suffix sum from t on
        const float incl = wave_incl_sum(val);
        __syncthreads();   // wsum of the previous block is consumed
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        float before = 0.0f, total = 0.0f;
#pragma unroll
        for (int w = 0; w < kGT / 64; ++w) {
            if (w < wave) before += wsum[w];
            total += wsum[w];
        }
        const float suffix = total - (before + incl) + val;
        if (t < T) {
            const float f = A.fpre[st + t];
            const double da = carry + static_cast<double>(suffix);
            A.dfp[st + t] = (f == -INFINITY) ? 0.0f : static_cast<float>(da / (1.0 + exp(static_cast<double>(f))));
            A.dip[st + t] = ci;
        }
        carry += static_cast<double>(total);
    }
    if (A.dm0 && tid == 0) {
        float dm = 0.0f;
        for (int b = 0; b < kScanBlocks; ++b) dm += A.dmp[static_cast<int64_t>(s) * kScanBlocks + b];
        A.dm0[s] = dm;
    }
}

// T = 0: the initial-state gradients are zero
__global__ void __launch_bounds__(256) bwd_zero_state_kernel(float* dC0, float* dn0, float* dm0, int S) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < static_cast<int64_t>(S) * kCV) dC0[i] = 0.0f;
    if (i < static_cast<int64_t>(S) * kDQK) dn0[i] = 0.0f;
    if (i < S) dm0[i] = 0.0f;
}

template <class Smem>
hipError_t launch_big(const void* kern, const BwdParams& p, unsigned grid, hipStream_t stream,
                      std::atomic<uint64_t>& raised, int threads = kBT) {
    const size_t lds = sizeof(Smem);
    hipError_t e = raise_dynamic_lds(kern, lds, raised);
    if (e != hipSuccess) return e;
    void* args[] = {const_cast<BwdParams*>(&p)};
    return hipLaunchKernel(kern, dim3(grid), dim3(threads), args, lds, stream);
}

size_t align256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

struct BwdLayout {
    size_t slots, seg, xp, hl, lz0, gamn, tok, part, chunk, dmp, total;
};
BwdLayout bwd_layout(int64_t S, int T) {
    const int64_t NC = (T + kBL - 1) / kBL, NC1 = NC > 0 ? NC - 1 : 0;
    BwdLayout L{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off += align256(bytes);
        return o;
    };
    L.slots = take(static_cast<size_t>(S * NC1 * kSlotFloats) * 4);
    L.seg = take(bwd_walk_workspace_bytes(S, T));
    L.xp = take(static_cast<size_t>(4 * S * T * kDQK) * 4);
    L.hl = take(static_cast<size_t>(S * NC1 * kCV) * 2);
    L.lz0 = take(static_cast<size_t>(S * kLzFloats) * 4);
    L.gamn = take(static_cast<size_t>(S * NC * kDQK) * 4);
    L.tok = take(static_cast<size_t>(S * T * kTokF) * 4);
    L.part = take(static_cast<size_t>(S * T * kPartF) * 4);
    L.chunk = take(static_cast<size_t>(S * NC) * 4);
    L.dmp = take(static_cast<size_t>(S * kScanBlocks) * 4);
    L.total = off;
    return L;
}

}  // namespace

bool chunk_bwd_supported(mlstm_dtype dt, int DQK, int DV, int L) {
    return dt == MLSTM_BF16 && DQK == kDQK && DV == kDV && L == kBL;
}

size_t chunk_bwd_workspace_bytes(int B, int NH, int T) {
    return bwd_layout(static_cast<int64_t>(B) * NH, T).total;
}

hipError_t launch_chunk_bwd(const ChunkBwdArgs& a, void* workspace, hipStream_t stream) {
    const int S = a.f.B * a.f.NH, T = a.f.T;
    if (S == 0) return hipSuccess;
    if (T == 0) {
        if (a.dC0) {
            const int64_t n = static_cast<int64_t>(S) * kCV;
            hipLaunchKernelGGL(bwd_zero_state_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream,
                               a.dC0, a.dn0, a.dm0, S);
            return hipGetLastError();
        }
        return hipSuccess;
    }
    const BwdLayout L = bwd_layout(S, T);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    BwdParams p{};
    p.q = static_cast<const uint16_t*>(a.f.q);
    p.k = static_cast<const uint16_t*>(a.f.k);
    p.v = static_cast<const uint16_t*>(a.f.v);
    p.dh = static_cast<const uint16_t*>(a.dh);
    p.ipre = a.f.ipre;
    p.fpre = a.f.fpre;
    p.C0 = a.f.C0;
    p.n0 = a.f.n0;
    p.m0 = a.f.m0;
    p.dq = a.dq;
    p.dk = a.dk;
    p.dv = a.dv;
    p.dip = a.dipre;
    p.dfp = a.dfpre;
    p.dC0 = a.dC0;
    p.dn0 = a.dn0;
    p.dm0 = a.dm0;
    p.slots = reinterpret_cast<float*>(ws + L.slots);
    p.hl = reinterpret_cast<uint16_t*>(ws + L.hl);
    p.lz0 = reinterpret_cast<float*>(ws + L.lz0);
    p.gamn = reinterpret_cast<float*>(ws + L.gamn);
    p.tok = reinterpret_cast<float*>(ws + L.tok);
    p.part = reinterpret_cast<float*>(ws + L.part);
    p.chunk = reinterpret_cast<float*>(ws + L.chunk);
    p.dmp = reinterpret_cast<float*>(ws + L.dmp);
    p.T = T;
    p.NC = (T + kBL - 1) / kBL;

    float* X = reinterpret_cast<float*>(ws + L.xp);
    hipError_t e = launch_bwd_walk(a.f, a.dh, p.slots, reinterpret_cast<float*>(ws + L.seg), X, p.part, stream);
    if (e != hipSuccess) return e;
    const int64_t n4 = static_cast<int64_t>(S) * T * kDQK / 4;
    hipLaunchKernelGGL(bwd_xsum_kernel, dim3(static_cast<unsigned>((n4 + 255) / 256)), dim3(256), 0, stream, X, a.dq, n4);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned nchunks = static_cast<unsigned>(S) * p.NC;
    static std::atomic<uint64_t> r_intra{0}, r_kv{0};
    e = launch_big<IntraSmem>(reinterpret_cast<const void*>(bwd_intra_kernel), p, nchunks, stream, r_intra);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bwd_scan_kernel, dim3(kScanBlocks, S), dim3(256), 0, stream, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_big<InterKVSmem>(reinterpret_cast<const void*>(bwd_interkv_kernel), p, nchunks, stream, r_kv, kIKT);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bwd_gate_kernel, dim3(S), dim3(kGT), 0, stream, p);
    return hipGetLastError();
}

#ifdef MLSTM_DEBUG
MLSTM_DEBUG_READER(debug_flags_chunk_bwd)
#endif

}  // namespace mlstm
