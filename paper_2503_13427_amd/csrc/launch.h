// Internal launch interface between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

#include "mlstm.h"

namespace mlstm {

// Raises a kernel's dynamic LDS limit to `bytes` on the current device, once per device;
// `done` is that kernel's mask of devices already raised (devices 64 and up are raised on
// every call).  Safe to call from several host threads: the attribute call is idempotent.
inline hipError_t raise_dynamic_lds(const void* kernel, size_t bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = dev < 64 ? (uint64_t{1} << dev) : 0;
    if (bit != 0 && (done.load(std::memory_order_acquire) & bit) != 0) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
    if (e == hipSuccess && bit != 0) done.fetch_or(bit, std::memory_order_release);
    return e;
}

// --- decode step -----------------------------------------------------------
hipError_t launch_step(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                       const float* fpre, const float* C, const float* n, const float* m, int B, int NH,
                       int DQK, int DV, void* h, float* C_out, float* n_out, float* m_out,
                       hipStream_t stream);
size_t step_lds_bytes(int DQK, int DV);
// the step with the output gate and headwise norm of the cell's output (fused when one workgroup
// owns each sequence's row, else the step and then the output pass in place)
bool step_output_fused(int B, int NH, int DQK, int DV);
hipError_t launch_step_output(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                              const float* fpre, const float* C, const float* n, const float* m, const void* o_pre,
                              const float* weight, const float* bias, float eps, int rms, int B, int NH, int DQK,
                              int DV, void* h, float* C_out, float* n_out, float* m_out, hipStream_t stream);

// --- hidden-state output: output gate and headwise norm ----------------------
constexpr int kOutNormMaxDV = 2048;
// element offset of row (b, head, t) is b * b + head * h + t * t; a row is DV contiguous elements
struct RowStrides {
    int64_t b, h, t;
};
hipError_t launch_output_norm(mlstm_dtype dt, const void* h_tilde, const void* o_pre, const float* weight,
                              const float* bias, float eps, int rms, int64_t rows, int NH, int T, int DV, void* h,
                              RowStrides so, RowStrides sy,
                              hipStream_t stream);

// --- gate pre-activations of a layer (bf16 x, W^T [2 NH, d]) -----------------
constexpr int kGateMaxCols = 64;   // 2 NH
constexpr int kGateDMultiple = 128;
hipError_t launch_gate_preact(const void* x, const void* w_t, const float* bias, float cap, const uint8_t* border,
                              int B, int T, int d, int NH, float* ipre, float* fpre, hipStream_t stream);

// --- backward pass over the parallel form (fp32 VALU) ------------------------
bool parallel_bwd_supported(int DQK, int DV);
size_t parallel_bwd_workspace_bytes(int B, int NH, int T, int DV);
hipError_t launch_parallel_bwd(mlstm_dtype dt, const void* q, const void* k, const void* v, const float* ipre,
                               const float* fpre, const float* dh, int B, int NH, int T, int DQK, int DV, float* dq,
                               float* dk, float* dv, float* dipre, float* dfpre, void* workspace, hipStream_t stream);

// --- chunkwise prefill, fp32 VALU kernel (small heads) -----------------------
struct ChunkArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* ipre;
    const float* fpre;
    const float* C0;  // may be NULL (zero state)
    const float* n0;
    const float* m0;
    int B, NH, T, DQK, DV, L;
    void* h;
    float* CT;
    float* nT;
    float* mT;
    // q, k, v element strides (batch, head, token) x 3, rows of D contiguous; NULL: contiguous
    // [B, NH, T, D] (the bf16 MFMA path reads them; the other kernels take contiguous rows only)
    const int64_t* strides = nullptr;
};

// Returns the dv tile the fp32 kernel would use, or 0 if no tile fits its LDS budget.
int chunk_f32_tile(int DQK, int DV, int L);
hipError_t launch_chunk_f32(mlstm_dtype dt, const ChunkArgs& a, hipStream_t stream);

// --- chunkwise prefill, bf16 MFMA kernels (DQK = 256, DV = 512) --------------
bool chunk_mfma_supported(mlstm_dtype dt, int DQK, int DV, int L);
// Number of sequence segments the segment-parallel schedule uses (1 = fused single pass).
int chunk_mfma_segments(int B, int NH, int T, int L);
size_t chunk_mfma_workspace_bytes(int B, int NH, int T, int DQK, int DV, int L);
hipError_t launch_chunk_mfma(const ChunkArgs& a, void* workspace, size_t workspace_bytes, hipStream_t stream);
// The prefill's segment schedule for chunks of L tokens: the segment count G (1: one segment per
// sequence), local sub-segments R per segment and chunks per segment.  launch_segment_states runs,
// when G > 1, the local pass (bf16 hi + lo products when hilo) and the combine into the segment slots
// ``seg`` (chunk_mfma_workspace_bytes of them).
struct SegmentShape {
    int G, R, seg_chunks;
};
SegmentShape segment_shape(int B, int NH, int T, int L, bool use_segments);
hipError_t launch_segment_states(const ChunkArgs& a, int L, const SegmentShape& sh, float* seg, bool hilo,
                                 hipStream_t stream);
// --- chunkwise backward (bf16, DQK = 256, DV = 512, L = 64) --------------------
bool chunk_bwd_supported(mlstm_dtype dt, int DQK, int DV, int L);
size_t chunk_bwd_workspace_bytes(int B, int NH, int T);
struct ChunkBwdArgs {
    ChunkArgs f;             // forward inputs (q, k, v, gates, initial state), sizes, L
    const void* dh;          // [B, NH, T, DV] (dt)
    float* dq;
    float* dk;
    float* dv;
    float* dipre;
    float* dfpre;
    float* dC0;              // NULL: the initial-state gradients are not wanted
    float* dn0;
    float* dm0;
};
hipError_t launch_chunk_bwd(const ChunkBwdArgs& a, void* workspace, hipStream_t stream);

// Fixed device scratch of mlstm_chunkwise_fwd_noalloc: a file-scope device array of this many bytes,
// one copy per device.  chunk_scratch gives its address on the current device (looked up once per
// device, then cached).
constexpr size_t kChunkScratchBytes = size_t(64) << 20;
hipError_t chunk_scratch(void** ptr);

#ifdef MLSTM_DEBUG
// Debug builds: each source file's bounds-check flag word, ORed into *out and cleared.
hipError_t debug_flags_chunk_mfma(unsigned int* out);
hipError_t debug_flags_chunk_f32(unsigned int* out);
hipError_t debug_flags_step(unsigned int* out);
hipError_t debug_flags_output_norm(unsigned int* out);
hipError_t debug_flags_gate_preact(unsigned int* out);
hipError_t debug_flags_chunk_bwd(unsigned int* out);
hipError_t debug_flags_parallel_bwd(unsigned int* out);
#endif

}  // namespace mlstm
