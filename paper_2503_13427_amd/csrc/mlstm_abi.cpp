// C-ABI layer of libmlstm: argument validation (pure host code, no HIP call
// before a call is accepted), kernel selection and launch.
#include <stdint.h>
#include <string.h>

#include <hip/hip_runtime.h>

#include "launch.h"
#include "mlstm.h"

namespace {

struct Range {
    uintptr_t lo, hi;  // [lo, hi)
};

inline Range range_of(const void* p, size_t bytes) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    return Range{a, a + bytes};
}

inline bool overlap(Range a, Range b) {
    if (a.lo == a.hi || b.lo == b.hi) return false;
    return a.lo < b.hi && b.lo < a.hi;
}

inline bool misaligned(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u); }

inline bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > INT64_MAX / a) return false;
    *out = a * b;
    return true;
}

// A C caller may pass any int as an mlstm_dtype: every test of the argument reads its raw value (a C++ enum
// load outside the enumerators' range is undefined behaviour).
// (reading the argument by value is such a load too, so these take its address)
inline int dtype_code(const mlstm_dtype* d) {
    int v;
    memcpy(&v, d, sizeof v);
    return v;
}
inline bool dtype_valid(const mlstm_dtype* d) { return dtype_code(d) == MLSTM_F32 || dtype_code(d) == MLSTM_BF16; }
inline int norm_code(const mlstm_norm* n) {
    int v;
    memcpy(&v, n, sizeof v);
    return v;
}
inline size_t elem_bytes(mlstm_dtype dt) { return dt == MLSTM_BF16 ? 2 : 4; }   // a validated dtype

}  // namespace

extern "C" {

const char* mlstm_status_string(mlstm_status s) {
    // a C caller may pass any int: read the raw value (an enum load outside its range is undefined in C++)
    int code;
    memcpy(&code, &s, sizeof code);
    switch (code) {
        case MLSTM_OK: return "MLSTM_OK";
        case MLSTM_ERR_NULL_PTR: return "MLSTM_ERR_NULL_PTR: a required pointer is NULL, or the initial state is partially given";
        case MLSTM_ERR_BAD_SHAPE: return "MLSTM_ERR_BAD_SHAPE: invalid size";
        case MLSTM_ERR_UNSUPPORTED: return "MLSTM_ERR_UNSUPPORTED: this (dtype, DQK, DV, L) combination is not built";
        case MLSTM_ERR_MISALIGNED: return "MLSTM_ERR_MISALIGNED: a tensor pointer is not 16-byte aligned";
        case MLSTM_ERR_ALIAS: return "MLSTM_ERR_ALIAS: an output overlaps an input or another output";
        case MLSTM_ERR_WORKSPACE:
            return "MLSTM_ERR_WORKSPACE: workspace smaller than the call's *_workspace_bytes, or (no-allocation "
                   "variant) more than the library's fixed scratch of mlstm_chunkwise_scratch_bytes";
        case MLSTM_ERR_HIP: return "MLSTM_ERR_HIP: the HIP runtime reported an error at launch";
    }
    return "MLSTM_UNKNOWN_STATUS";
}

int mlstm_version(void) { return 100; }

unsigned int mlstm_debug_flags(void) {
#ifdef MLSTM_DEBUG
    unsigned int f = 0;
    hipError_t (*const readers[])(unsigned int*) = {
        mlstm::debug_flags_chunk_mfma, mlstm::debug_flags_chunk_f32,  mlstm::debug_flags_step,
        mlstm::debug_flags_output_norm, mlstm::debug_flags_gate_preact, mlstm::debug_flags_chunk_bwd,
        mlstm::debug_flags_parallel_bwd};
    for (auto r : readers)
        if (r(&f) != hipSuccess) return MLSTM_DEBUG_NOT_BUILT | 0x40000000u;   // the words could not be read
    return f;
#else
    return MLSTM_DEBUG_NOT_BUILT;
#endif
}

size_t mlstm_chunkwise_workspace_bytes(int B, int NH, int T, int DQK, int DV, int L, mlstm_dtype dt) {
    if (B <= 0 || NH <= 0 || T < 0 || L <= 0 || !dtype_valid(&dt)) return 0;
    if (!mlstm::chunk_mfma_supported(dt, DQK, DV, L)) return 0;
    return mlstm::chunk_mfma_workspace_bytes(B, NH, T, DQK, DV, L);
}

// Validation and launch shared by mlstm_chunkwise_fwd (caller workspace) and
// mlstm_chunkwise_fwd_noalloc (the library's fixed device scratch, use_scratch) and
// mlstm_chunkwise_fwd_strided (strides: q, k, v element strides, else NULL for contiguous rows).
static mlstm_status chunkwise_fwd_impl(const void* q, const void* k, const void* v, const int64_t* strides, int dtc,
                                       const float* ipre, const float* fpre, const float* C0, const float* n0,
                                       const float* m0, int B, int NH, int T, int DQK, int DV, int L, void* h,
                                       float* CT, float* nT, float* mT, void* workspace, size_t workspace_bytes,
                                       bool use_scratch, void* hip_stream) {
    // per-token buffers are empty (and may be NULL) when T == 0
    if (T != 0 && (!q || !k || !v || !ipre || !fpre || !h)) return MLSTM_ERR_NULL_PTR;
    if (!CT || !nT || !mT) return MLSTM_ERR_NULL_PTR;
    const int n_init = (C0 != nullptr) + (n0 != nullptr) + (m0 != nullptr);
    if (n_init != 0 && n_init != 3) return MLSTM_ERR_NULL_PTR;
    if (workspace_bytes > 0 && !workspace) return MLSTM_ERR_NULL_PTR;
    if (dtc != MLSTM_F32 && dtc != MLSTM_BF16) return MLSTM_ERR_UNSUPPORTED;
    const mlstm_dtype dt = static_cast<mlstm_dtype>(dtc);
    if (B <= 0 || NH <= 0 || T < 0 || DQK <= 0 || DV <= 0 || L <= 0) return MLSTM_ERR_BAD_SHAPE;

    int64_t S, ST, nq, nv, nC, nn;
    if (!mul_ok(B, NH, &S) || !mul_ok(S, T, &ST) || !mul_ok(ST, DQK, &nq) || !mul_ok(ST, DV, &nv) ||
        !mul_ok(S, static_cast<int64_t>(DQK) * DV, &nC) || !mul_ok(S, DQK, &nn) || S > INT32_MAX)
        return MLSTM_ERR_BAD_SHAPE;

    const void* ptrs[] = {q, k, v, ipre, fpre, C0, n0, m0, h, CT, nT, mT, workspace};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;

    const size_t eb = elem_bytes(dt);
    // strided q, k, v: the element range each view spans (rows of D contiguous, every row 16-byte aligned)
    int64_t eq = nq, ek = nq, ev = nv;
    if (strides) {
        for (int i = 0; i < 9; ++i) {
            if (strides[i] < 0) return MLSTM_ERR_BAD_SHAPE;
            if (strides[i] % 8) return MLSTM_ERR_MISALIGNED;
        }
        if (strides[2] < DQK || strides[5] < DQK || strides[8] < DV) return MLSTM_ERR_BAD_SHAPE;   // rows overlap
        // the kernels split a sequence index into (batch, head) by a 32-bit reciprocal multiply
        if (static_cast<int64_t>(B) * NH * NH >= (int64_t(1) << 32)) return MLSTM_ERR_UNSUPPORTED;
        int64_t* ext[3] = {&eq, &ek, &ev};
        const int D[3] = {DQK, DQK, DV};
        for (int j = 0; j < 3; ++j) {
            const int64_t* x = strides + 3 * j;
            if (ST == 0) {
                *ext[j] = 0;
                continue;
            }
            if (x[0] > INT64_MAX / 4 / B || x[1] > INT64_MAX / 4 / NH || x[2] > INT64_MAX / 4 / T)
                return MLSTM_ERR_BAD_SHAPE;
            *ext[j] = (B - 1) * x[0] + (NH - 1) * x[1] + (static_cast<int64_t>(T) - 1) * x[2] + D[j];
            // one sequence's rows are addressed through a 32-bit buffer offset, including the up to 127
            // rows past its end that a partial last chunk reads (as zeros, outside the buffer range)
            if (((static_cast<int64_t>(T) + 127) * x[2] + D[j]) * 2 >= (int64_t(1) << 31)) return MLSTM_ERR_UNSUPPORTED;
        }
    }
    const Range in[] = {range_of(q, eq * eb), range_of(k, ek * eb), range_of(v, ev * eb),
                        range_of(ipre, ST * 4), range_of(fpre, ST * 4), range_of(C0, C0 ? nC * 4 : 0),
                        range_of(n0, n0 ? nn * 4 : 0), range_of(m0, m0 ? S * 4 : 0)};
    const Range out[] = {range_of(h, nv * eb), range_of(CT, nC * 4), range_of(nT, nn * 4), range_of(mT, S * 4),
                         range_of(workspace, workspace_bytes)};
    for (const Range& o : out) {
        for (const Range& i : in)
            if (overlap(o, i)) return MLSTM_ERR_ALIAS;
    }
    for (size_t a = 0; a < sizeof(out) / sizeof(out[0]); ++a)
        for (size_t b = a + 1; b < sizeof(out) / sizeof(out[0]); ++b)
            if (overlap(out[a], out[b])) return MLSTM_ERR_ALIAS;

    const bool mfma = mlstm::chunk_mfma_supported(dt, DQK, DV, L);
    if (!mfma && (strides || mlstm::chunk_f32_tile(DQK, DV, L) == 0)) return MLSTM_ERR_UNSUPPORTED;
    // the MFMA kernel addresses one sequence's v through a 32-bit buffer range
    if (mfma && static_cast<int64_t>(T) * DV * 2 >= (int64_t(1) << 31)) return MLSTM_ERR_UNSUPPORTED;

    size_t ws_need = 0;
    if (mfma) ws_need = mlstm::chunk_mfma_workspace_bytes(B, NH, T, DQK, DV, L);
    if (workspace_bytes > 0 && workspace_bytes < ws_need) return MLSTM_ERR_WORKSPACE;
    if (use_scratch && ws_need > mlstm::kChunkScratchBytes) return MLSTM_ERR_WORKSPACE;

    mlstm::ChunkArgs a{q, k, v, ipre, fpre, C0, n0, m0, B, NH, T, DQK, DV, L, h, CT, nT, mT, strides};
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    if (use_scratch && ws_need > 0) {
        hipError_t e = mlstm::chunk_scratch(&workspace);
        if (e != hipSuccess) return MLSTM_ERR_HIP;
        workspace_bytes = ws_need;
    }
    hipError_t e = mfma ? mlstm::launch_chunk_mfma(a, workspace_bytes ? workspace : nullptr,
                                                   workspace_bytes, stream)
                        : mlstm::launch_chunk_f32(dt, a, stream);
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

mlstm_status mlstm_chunkwise_fwd(const void* q, const void* k, const void* v, mlstm_dtype dt,
                                 const float* ipre, const float* fpre, const float* C0, const float* n0,
                                 const float* m0, int B, int NH, int T, int DQK, int DV, int L, void* h,
                                 float* CT, float* nT, float* mT, void* workspace, size_t workspace_bytes,
                                 void* hip_stream) {
    return chunkwise_fwd_impl(q, k, v, nullptr, dtype_code(&dt), ipre, fpre, C0, n0, m0, B, NH, T, DQK, DV, L, h, CT,
                              nT, mT, workspace, workspace_bytes, false, hip_stream);
}

mlstm_status mlstm_chunkwise_fwd_strided(const void* q, const void* k, const void* v, const int64_t* qkv_strides,
                                         mlstm_dtype dt, const float* ipre, const float* fpre, const float* C0,
                                         const float* n0, const float* m0, int B, int NH, int T, int DQK, int DV,
                                         int L, void* h, float* CT, float* nT, float* mT, void* workspace,
                                         size_t workspace_bytes, void* hip_stream) {
    if (!qkv_strides) return MLSTM_ERR_NULL_PTR;
    return chunkwise_fwd_impl(q, k, v, qkv_strides, dtype_code(&dt), ipre, fpre, C0, n0, m0, B, NH, T, DQK, DV, L, h,
                              CT, nT, mT, workspace, workspace_bytes, false, hip_stream);
}

size_t mlstm_chunkwise_scratch_bytes(void) { return mlstm::kChunkScratchBytes; }

mlstm_status mlstm_chunkwise_fwd_noalloc(const void* q, const void* k, const void* v, mlstm_dtype dt,
                                         const float* ipre, const float* fpre, const float* C0, const float* n0,
                                         const float* m0, int B, int NH, int T, int DQK, int DV, int L, void* h,
                                         float* CT, float* nT, float* mT, void* hip_stream) {
    return chunkwise_fwd_impl(q, k, v, nullptr, dtype_code(&dt), ipre, fpre, C0, n0, m0, B, NH, T, DQK, DV, L, h, CT,
                              nT, mT, nullptr, 0, true, hip_stream);
}

// Validation shared by mlstm_step and mlstm_step_output (extra: the o~, weight and bias ranges
// of the output variant, which h may not overlap either).
static mlstm_status step_validate(const void* q, const void* k, const void* v, int dtc, const float* ipre,
                                  const float* fpre, const float* C, const float* n, const float* m, int B, int NH,
                                  int DQK, int DV, void* h, float* C_out, float* n_out, float* m_out,
                                  const Range* extra, int n_extra) {
    if (!q || !k || !v || !ipre || !fpre || !C || !n || !m || !h || !C_out || !n_out || !m_out)
        return MLSTM_ERR_NULL_PTR;
    if (dtc != MLSTM_F32 && dtc != MLSTM_BF16) return MLSTM_ERR_UNSUPPORTED;
    const mlstm_dtype dt = static_cast<mlstm_dtype>(dtc);
    if (B <= 0 || NH <= 0 || DQK <= 0 || DV <= 0 || (DV % 4)) return MLSTM_ERR_BAD_SHAPE;
    if (static_cast<int64_t>(DQK) * DV > (int64_t(1) << 20) || DQK > 4096) return MLSTM_ERR_UNSUPPORTED;
    int64_t S;
    if (!mul_ok(B, NH, &S) || S > INT32_MAX) return MLSTM_ERR_BAD_SHAPE;

    const void* ptrs[] = {q, k, v, ipre, fpre, C, n, m, h, C_out, n_out, m_out};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;

    const size_t eb = elem_bytes(dt);
    const int64_t nC = S * DQK * DV, nn = S * DQK;
    const Range rq = range_of(q, S * DQK * eb), rk = range_of(k, S * DQK * eb), rv = range_of(v, S * DV * eb);
    const Range ri = range_of(ipre, S * 4), rf = range_of(fpre, S * 4);
    const Range rC = range_of(C, nC * 4), rn = range_of(n, nn * 4), rm = range_of(m, S * 4);
    const Range rh = range_of(h, S * DV * eb), rCo = range_of(C_out, nC * 4), rno = range_of(n_out, nn * 4),
                rmo = range_of(m_out, S * 4);
    // h overlaps nothing
    for (const Range& r : {rq, rk, rv, ri, rf, rC, rn, rm, rCo, rno, rmo})
        if (overlap(rh, r)) return MLSTM_ERR_ALIAS;
    for (int i = 0; i < n_extra; ++i)
        if (overlap(rh, extra[i])) return MLSTM_ERR_ALIAS;
    // each state output may equal its own input exactly, and overlaps nothing else
    struct Pair {
        Range out;
        Range same;
        bool exact;
    };
    const Pair pairs[] = {{rCo, rC, C_out == C}, {rno, rn, n_out == n}, {rmo, rm, m_out == m}};
    for (const Pair& p : pairs) {
        if (overlap(p.out, p.same) && !p.exact) return MLSTM_ERR_ALIAS;
        for (const Range& r : {rq, rk, rv, ri, rf})
            if (overlap(p.out, r)) return MLSTM_ERR_ALIAS;
        for (int i = 0; i < n_extra; ++i)
            if (overlap(p.out, extra[i])) return MLSTM_ERR_ALIAS;
    }
    if (overlap(rCo, rn) || overlap(rCo, rm) || overlap(rno, rC) || overlap(rno, rm) || overlap(rmo, rC) ||
        overlap(rmo, rn) || overlap(rCo, rno) || overlap(rCo, rmo) || overlap(rno, rmo))
        return MLSTM_ERR_ALIAS;
    return MLSTM_OK;
}

mlstm_status mlstm_step(const void* q, const void* k, const void* v, mlstm_dtype dt, const float* ipre,
                        const float* fpre, const float* C, const float* n, const float* m, int B, int NH,
                        int DQK, int DV, void* h, float* C_out, float* n_out, float* m_out,
                        void* hip_stream) {
    const mlstm_status st = step_validate(q, k, v, dtype_code(&dt), ipre, fpre, C, n, m, B, NH, DQK, DV, h, C_out, n_out, m_out,
                                          nullptr, 0);
    if (st != MLSTM_OK) return st;
    hipError_t e = mlstm::launch_step(dt, q, k, v, ipre, fpre, C, n, m, B, NH, DQK, DV, h, C_out, n_out, m_out,
                                      static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

mlstm_status mlstm_step_output(const void* q, const void* k, const void* v, mlstm_dtype dt, const float* ipre,
                               const float* fpre, const float* C, const float* n, const float* m,
                               const void* o_pre, const float* weight, const float* bias, float eps,
                               mlstm_norm norm, int B, int NH, int DQK, int DV, void* h, float* C_out,
                               float* n_out, float* m_out, void* hip_stream) {
    if (!o_pre) return MLSTM_ERR_NULL_PTR;
    if (!(eps > 0.0f) || eps > 3.0e38f) return MLSTM_ERR_BAD_SHAPE;   // rejects NaN and inf too
    if (norm_code(&norm) != MLSTM_NORM_LAYER && norm_code(&norm) != MLSTM_NORM_RMS) return MLSTM_ERR_BAD_SHAPE;
    if (B > 0 && NH > 0 && DV > mlstm::kOutNormMaxDV) return MLSTM_ERR_UNSUPPORTED;
    if (misaligned(o_pre) || misaligned(weight) || misaligned(bias)) return MLSTM_ERR_MISALIGNED;
    int64_t S = 0, nw = 0;
    if (!mul_ok(B, NH, &S) || !mul_ok(NH, DV, &nw)) return MLSTM_ERR_BAD_SHAPE;
    if (!dtype_valid(&dt)) return MLSTM_ERR_UNSUPPORTED;
    const Range extra[] = {range_of(o_pre, S * DV * elem_bytes(dt)), range_of(weight, weight ? nw * 4 : 0),
                           range_of(bias, bias ? nw * 4 : 0)};
    const mlstm_status st = step_validate(q, k, v, dtype_code(&dt), ipre, fpre, C, n, m, B, NH, DQK, DV, h, C_out, n_out, m_out,
                                          extra, 3);
    if (st != MLSTM_OK) return st;
    hipError_t e = mlstm::launch_step_output(dt, q, k, v, ipre, fpre, C, n, m, o_pre, weight, bias, eps,
                                             norm == MLSTM_NORM_RMS, B, NH, DQK, DV, h, C_out, n_out, m_out,
                                             static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

mlstm_status mlstm_output_norm(const void* h_tilde, const void* o_pre, mlstm_dtype dt, const float* weight,
                               const float* bias, float eps, mlstm_norm norm, int B, int NH, int T, int DV,
                               void* h, void* hip_stream) {
    if (T != 0 && (!h_tilde || !o_pre || !h)) return MLSTM_ERR_NULL_PTR;
    if (!dtype_valid(&dt)) return MLSTM_ERR_UNSUPPORTED;
    if (B <= 0 || NH <= 0 || T < 0 || DV <= 0) return MLSTM_ERR_BAD_SHAPE;
    if (!(eps > 0.0f) || eps > 3.0e38f) return MLSTM_ERR_BAD_SHAPE;   // rejects NaN and inf too
    if (norm_code(&norm) != MLSTM_NORM_LAYER && norm_code(&norm) != MLSTM_NORM_RMS) return MLSTM_ERR_BAD_SHAPE;
    if ((DV % 4) || DV > mlstm::kOutNormMaxDV) return MLSTM_ERR_UNSUPPORTED;
    int64_t S, rows, nel, nw;
    if (!mul_ok(B, NH, &S) || !mul_ok(S, T, &rows) || !mul_ok(rows, DV, &nel) || !mul_ok(NH, DV, &nw) ||
        rows / 4 >= INT32_MAX)
        return MLSTM_ERR_BAD_SHAPE;
    const void* ptrs[] = {h_tilde, o_pre, weight, bias, h};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;
    const size_t eb = elem_bytes(dt);
    const Range rx = range_of(h_tilde, nel * eb), ro = range_of(o_pre, nel * eb), rh = range_of(h, nel * eb);
    const Range rw = range_of(weight, weight ? nw * 4 : 0), rb = range_of(bias, bias ? nw * 4 : 0);
    // h may be h_tilde exactly (in place) and overlaps nothing else
    if ((overlap(rh, rx) && h != h_tilde) || overlap(rh, ro) || overlap(rh, rw) || overlap(rh, rb))
        return MLSTM_ERR_ALIAS;
    if (rows == 0) return MLSTM_OK;
    const mlstm::RowStrides hm{static_cast<int64_t>(NH) * T * DV, static_cast<int64_t>(T) * DV, DV};
    hipError_t e = mlstm::launch_output_norm(dt, h_tilde, o_pre, weight, bias, eps, norm == MLSTM_NORM_RMS, rows, NH,
                                             T, DV, h, hm, hm, static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

mlstm_status mlstm_output_norm_tokens(const void* h_tilde, const void* o_pre, int64_t o_token_stride, mlstm_dtype dt,
                                      const float* weight, const float* bias, float eps, mlstm_norm norm, int B,
                                      int NH, int T, int DV, void* y, void* hip_stream) {
    if (T != 0 && (!h_tilde || !o_pre || !y)) return MLSTM_ERR_NULL_PTR;
    if (!dtype_valid(&dt)) return MLSTM_ERR_UNSUPPORTED;
    if (B <= 0 || NH <= 0 || T < 0 || DV <= 0) return MLSTM_ERR_BAD_SHAPE;
    if (!(eps > 0.0f) || eps > 3.0e38f) return MLSTM_ERR_BAD_SHAPE;
    if (norm_code(&norm) != MLSTM_NORM_LAYER && norm_code(&norm) != MLSTM_NORM_RMS) return MLSTM_ERR_BAD_SHAPE;
    if ((DV % 4) || DV > mlstm::kOutNormMaxDV) return MLSTM_ERR_UNSUPPORTED;
    int64_t S, rows, nel, nw, toks, ospan;
    if (!mul_ok(B, NH, &S) || !mul_ok(S, T, &rows) || !mul_ok(rows, DV, &nel) || !mul_ok(NH, DV, &nw) ||
        !mul_ok(B, T, &toks) || rows / 4 >= INT32_MAX)
        return MLSTM_ERR_BAD_SHAPE;
    // o~ rows of one token may not overlap one another; the stride keeps rows DV-aligned like the others
    if (o_token_stride < nw || o_token_stride % 4) return MLSTM_ERR_BAD_SHAPE;
    if (toks > 0 && (!mul_ok(toks - 1, o_token_stride, &ospan) || ospan > INT64_MAX - nw)) return MLSTM_ERR_BAD_SHAPE;
    const void* ptrs[] = {h_tilde, o_pre, weight, bias, y};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;
    const size_t eb = elem_bytes(dt);
    const int64_t oel = toks > 0 ? ospan + nw : 0;
    const Range rx = range_of(h_tilde, nel * eb), ro = range_of(o_pre, oel * eb), ry = range_of(y, nel * eb);
    const Range rw = range_of(weight, weight ? nw * 4 : 0), rb = range_of(bias, bias ? nw * 4 : 0);
    if (overlap(ry, rx) || overlap(ry, ro) || overlap(ry, rw) || overlap(ry, rb)) return MLSTM_ERR_ALIAS;
    if (rows == 0) return MLSTM_OK;
    const mlstm::RowStrides so{static_cast<int64_t>(T) * o_token_stride, DV, o_token_stride};
    const mlstm::RowStrides sy{static_cast<int64_t>(T) * NH * DV, DV, static_cast<int64_t>(NH) * DV};
    hipError_t e = mlstm::launch_output_norm(dt, h_tilde, o_pre, weight, bias, eps, norm == MLSTM_NORM_RMS, rows, NH,
                                             T, DV, y, so, sy, static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

mlstm_status mlstm_gate_preact(const void* x, mlstm_dtype dt, const void* w_t, const float* bias, float cap,
                               const unsigned char* border, int B, int T, int d, int NH, float* ipre, float* fpre,
                               void* hip_stream) {
    if (B < 0 || T < 0 || d <= 0 || NH <= 0) return MLSTM_ERR_BAD_SHAPE;
    int64_t M, nx, ng, nw;
    if (!mul_ok(B, T, &M) || !mul_ok(M, d, &nx) || !mul_ok(M, NH, &ng) || !mul_ok(2 * static_cast<int64_t>(NH), d, &nw))
        return MLSTM_ERR_BAD_SHAPE;
    if (M != 0 && (!x || !w_t || !ipre || !fpre)) return MLSTM_ERR_NULL_PTR;
    if (!(cap >= 0.0f) || cap > 3.0e38f) return MLSTM_ERR_BAD_SHAPE;   // rejects NaN and inf too
    if (dtype_code(&dt) != MLSTM_BF16 || d % mlstm::kGateDMultiple || 2 * static_cast<int64_t>(NH) > mlstm::kGateMaxCols)
        return MLSTM_ERR_UNSUPPORTED;
    // a workgroup addresses its 64 rows of x, and all of w_t, through 32-bit byte offsets
    if (64 * static_cast<int64_t>(d) * 2 >= (int64_t(1) << 31) || nw * 2 >= (int64_t(1) << 31))
        return MLSTM_ERR_UNSUPPORTED;
    const void* ptrs[] = {x, w_t, bias, border, ipre, fpre};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;
    const Range rx = range_of(x, nx * 2), rw = range_of(w_t, nw * 2);
    const Range rb = range_of(bias, bias ? 2 * static_cast<size_t>(NH) * 4 : 0);
    const Range rd = range_of(border, border ? static_cast<size_t>(M) : 0);
    const Range ri = range_of(ipre, ng * 4), rf = range_of(fpre, ng * 4);
    if (overlap(ri, rf)) return MLSTM_ERR_ALIAS;
    for (const Range& o : {ri, rf})
        for (const Range& r : {rx, rw, rb, rd})
            if (overlap(o, r)) return MLSTM_ERR_ALIAS;
    if (M == 0) return MLSTM_OK;
    hipError_t e = mlstm::launch_gate_preact(x, w_t, bias, cap, border, B, T, d, NH, ipre, fpre,
                                             static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

size_t mlstm_parallel_bwd_workspace_bytes(int B, int NH, int T, int DV) {
    if (B <= 0 || NH <= 0 || T < 0 || DV <= 0) return 0;
    return mlstm::parallel_bwd_workspace_bytes(B, NH, T, DV);
}

mlstm_status mlstm_parallel_bwd(const void* q, const void* k, const void* v, mlstm_dtype dt, const float* ipre,
                                const float* fpre, const float* dh, int B, int NH, int T, int DQK, int DV, float* dq,
                                float* dk, float* dv, float* dipre, float* dfpre, void* workspace,
                                size_t workspace_bytes, void* hip_stream) {
    if (B <= 0 || NH <= 0 || T < 0 || DQK <= 0 || DV <= 0) return MLSTM_ERR_BAD_SHAPE;
    int64_t S, nt, nqk, nv;
    if (!mul_ok(B, NH, &S) || !mul_ok(S, T, &nt) || !mul_ok(nt, DQK, &nqk) || !mul_ok(nt, DV, &nv) ||
        S * ((static_cast<int64_t>(T) + 15) / 16) > INT32_MAX)
        return MLSTM_ERR_BAD_SHAPE;
    if (T != 0) {
        const void* req[] = {q, k, v, ipre, fpre, dh, dq, dk, dv, dipre, dfpre, workspace};
        for (const void* p : req)
            if (!p) return MLSTM_ERR_NULL_PTR;
    }
    if (!dtype_valid(&dt)) return MLSTM_ERR_UNSUPPORTED;
    if (!mlstm::parallel_bwd_supported(DQK, DV)) return MLSTM_ERR_UNSUPPORTED;
    const size_t ws_need = mlstm::parallel_bwd_workspace_bytes(B, NH, T, DV);
    if (T != 0 && workspace_bytes < ws_need) return MLSTM_ERR_WORKSPACE;
    const void* ptrs[] = {q, k, v, ipre, fpre, dh, dq, dk, dv, dipre, dfpre, workspace};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;
    const size_t eb = elem_bytes(dt);
    const Range ins[] = {range_of(q, nqk * eb), range_of(k, nqk * eb), range_of(v, nv * eb), range_of(ipre, nt * 4),
                         range_of(fpre, nt * 4), range_of(dh, nv * 4)};
    const Range outs[] = {range_of(dq, nqk * 4), range_of(dk, nqk * 4), range_of(dv, nv * 4),
                          range_of(dipre, nt * 4), range_of(dfpre, nt * 4), range_of(workspace, ws_need)};
    const size_t nouts = sizeof(outs) / sizeof(outs[0]);
    for (size_t a = 0; a < nouts; ++a) {
        for (const Range& r : ins)
            if (overlap(outs[a], r)) return MLSTM_ERR_ALIAS;
        for (size_t b = a + 1; b < nouts; ++b)
            if (overlap(outs[a], outs[b])) return MLSTM_ERR_ALIAS;
    }
    if (T == 0) return MLSTM_OK;
    hipError_t e = mlstm::launch_parallel_bwd(dt, q, k, v, ipre, fpre, dh, B, NH, T, DQK, DV, dq, dk, dv, dipre,
                                              dfpre, workspace, static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

size_t mlstm_chunkwise_bwd_workspace_bytes(int B, int NH, int T, int DQK, int DV, int L, mlstm_dtype dt) {
    if (B <= 0 || NH <= 0 || T < 0 || !dtype_valid(&dt) || !mlstm::chunk_bwd_supported(dt, DQK, DV, L)) return 0;
    return mlstm::chunk_bwd_workspace_bytes(B, NH, T);
}

mlstm_status mlstm_chunkwise_bwd(const void* q, const void* k, const void* v, mlstm_dtype dt, const float* ipre,
                                 const float* fpre, const float* C0, const float* n0, const float* m0, int B, int NH,
                                 int T, int DQK, int DV, int L, const void* dh, float* dq, float* dk,
                                 float* dv, float* dipre, float* dfpre, float* dC0, float* dn0, float* dm0,
                                 void* workspace, size_t workspace_bytes, void* hip_stream) {
    if (B <= 0 || NH <= 0 || T < 0 || DQK <= 0 || DV <= 0 || L <= 0) return MLSTM_ERR_BAD_SHAPE;
    if (T != 0) {
        const void* req[] = {q, k, v, ipre, fpre, dh, dq, dk, dv, dipre, dfpre, workspace};
        for (const void* p : req)
            if (!p) return MLSTM_ERR_NULL_PTR;
    }
    const int n_init = (C0 != nullptr) + (n0 != nullptr) + (m0 != nullptr);
    const int n_grad = (dC0 != nullptr) + (dn0 != nullptr) + (dm0 != nullptr);
    if ((n_init != 0 && n_init != 3) || (n_grad != 0 && n_grad != 3)) return MLSTM_ERR_NULL_PTR;
    if (!dtype_valid(&dt)) return MLSTM_ERR_UNSUPPORTED;
    int64_t S, nt, nqk, nv, nC, nn;
    if (!mul_ok(B, NH, &S) || !mul_ok(S, T, &nt) || !mul_ok(nt, DQK, &nqk) || !mul_ok(nt, DV, &nv) ||
        !mul_ok(S, static_cast<int64_t>(DQK) * DV, &nC) || !mul_ok(S, DQK, &nn))
        return MLSTM_ERR_BAD_SHAPE;
    if (!mlstm::chunk_bwd_supported(dt, DQK, DV, L)) return MLSTM_ERR_UNSUPPORTED;
    // one sequence's rows are addressed through 32-bit buffer ranges; the state scan has one grid row
    // per sequence; the chunk passes launch 4 workgroups per (sequence, chunk)
    if (static_cast<int64_t>(T) * DV * 2 >= (int64_t(1) << 31) || S > 65535 ||
        S * ((static_cast<int64_t>(T) + 63) / 64) * 4 > INT32_MAX)
        return MLSTM_ERR_UNSUPPORTED;
    const size_t ws_need = mlstm::chunk_bwd_workspace_bytes(B, NH, T);
    if (T != 0 && workspace_bytes < ws_need) return MLSTM_ERR_WORKSPACE;
    const void* ptrs[] = {q, k, v, ipre, fpre, C0, n0, m0, dh, dq, dk, dv, dipre, dfpre, dC0, dn0, dm0, workspace};
    for (const void* p : ptrs)
        if (misaligned(p)) return MLSTM_ERR_MISALIGNED;
    const size_t eb = elem_bytes(dt);
    const Range ins[] = {range_of(q, nqk * eb), range_of(k, nqk * eb), range_of(v, nv * eb), range_of(ipre, nt * 4),
                         range_of(fpre, nt * 4), range_of(C0, C0 ? nC * 4 : 0), range_of(n0, n0 ? nn * 4 : 0),
                         range_of(m0, m0 ? S * 4 : 0), range_of(dh, nv * eb)};
    const Range outs[] = {range_of(dq, nqk * 4), range_of(dk, nqk * 4), range_of(dv, nv * 4),
                          range_of(dipre, nt * 4), range_of(dfpre, nt * 4), range_of(dC0, dC0 ? nC * 4 : 0),
                          range_of(dn0, dn0 ? nn * 4 : 0), range_of(dm0, dm0 ? S * 4 : 0),
                          range_of(workspace, T != 0 ? ws_need : 0)};
    const size_t nouts = sizeof(outs) / sizeof(outs[0]);
    for (size_t a = 0; a < nouts; ++a) {
        for (const Range& r : ins)
            if (overlap(outs[a], r)) return MLSTM_ERR_ALIAS;
        for (size_t b = a + 1; b < nouts; ++b)
            if (overlap(outs[a], outs[b])) return MLSTM_ERR_ALIAS;
    }
    mlstm::ChunkBwdArgs a{};
    a.f = mlstm::ChunkArgs{q, k, v, ipre, fpre, C0, n0, m0, B, NH, T, DQK, DV, L, nullptr, nullptr, nullptr, nullptr};
    a.dh = dh;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.dipre = dipre;
    a.dfpre = dfpre;
    a.dC0 = dC0;
    a.dn0 = dn0;
    a.dm0 = dm0;
    hipError_t e = mlstm::launch_chunk_bwd(a, workspace, static_cast<hipStream_t>(hip_stream));
    return e == hipSuccess ? MLSTM_OK : MLSTM_ERR_HIP;
}

}  // extern "C"
