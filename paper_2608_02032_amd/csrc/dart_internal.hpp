// dart_internal.hpp -- launcher interface between the C ABI layer and the
// kernels.  Shapes are validated by the caller; launchers only enqueue.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dart {

struct Shape {
    int64_t B, L;
    int H, G, P, N, S;
    int64_t M;     // ceil(L/S)
    int64_t Mcap;  // memory slots
    int dtype;     // 0 fp32, 1 bf16
};

// Workspace of the scan: per-chunk log decay [B][H][M] (float), the
// chunk-entry states [B][M][H][N][P] (storage dtype), the within-chunk
// cumulative log decay [B][H][M][S] and the causal Gram tiles of every chunk
// and group (float).
size_t scan_workspace_bytes(const Shape& s);
hipError_t launch_scan(const Shape& s, const void* x, const float* dt, const float* A,
                       const void* Bm, const void* Cm, const float* h0, void* y_ssd, void* mem,
                       float* h_last, void* ws, hipStream_t st);

// The tuned kernels serve N in {32, 64, 128} with S in {64, 128, 256}; every
// other supported shape (N in {16, 32, 64, 128}, any S) takes the generic
// kernels of generic.hip.
bool tuned_shape(const Shape& s);

// Workspace pieces of the generic scan: per-chunk log decay [B][H][M], the
// chunk-entry states in the storage dtype (where the tuned scan keeps them),
// the chunk contributions and the entry states in float, [B][M][H][N][P].
struct GenScanWs {
    float* lda;
    void* states;
    float* dh32;
    float* st32;
};
hipError_t launch_gscan(const Shape& s, const void* x, const float* dt, const float* A,
                        const void* Bm, const void* Cm, const float* h0, void* y_ssd, void* mem,
                        float* h_last, const GenScanWs& w, hipStream_t st);

// The chunk-entry states H_[c-1] a scan left in its workspace,
// [B][M][H][N][P] in the storage dtype (H_[-1] = h0 or 0).
const void* scan_entry_states(const Shape& s, const void* ws);
// Every chunk's entry state in float for a backward pass: the chunk
// contributions dH32 [B][M][H][N][P] run token by token in float, the chunk
// log decays lda [B][H][M], and st32 [B][M][H][N][P] = H_[c-1] (h0 or 0 for
// c = 0), accumulated in float from dH32 -- the trajectory the backward's
// own token sweeps reproduce, so the decay gradient telescopes across chunk
// boundaries without a storage-dtype rounding at each.
hipError_t launch_scan_states_f32(const Shape& s, const void* x, const float* dt, const float* A,
                                  const void* Bm, const float* h0, float* lda, float* dh32,
                                  float* st32, hipStream_t st);

// Backward of the scan and its memories (scan_bwd.hip).
size_t ssd_bwd_workspace_bytes(const Shape& s);
hipError_t launch_ssd_bwd(const Shape& s, const void* x, const float* dt, const float* A,
                          const void* Bm, const void* Cm, const float* h0, const void* dy,
                          const float* dmem, const float* dh_last, float* dx, float* ddt, float* dA,
                          float* dB, float* dC, float* dh0, void* ws, hipStream_t st);

// The chunked-matrix scan backward on MFMA (scan_bwd_mfma.hip): bf16 storage
// and the tuned shapes; launch_ssd_bwd dispatches to it.
bool sbwd_mfma_shape(const Shape& s);
size_t sbwd_mfma_workspace_bytes(const Shape& s);
hipError_t launch_ssd_bwd_mfma(const Shape& s, const void* x, const float* dt, const float* A,
                               const void* Bm, const void* Cm, const float* h0, const void* dy,
                               const float* dmem, const float* dh_last, float* dx, float* ddt, float* dA,
                               float* dB, float* dC, float* dh0, void* ws, hipStream_t st);

struct SmaArgs {
    float eps;
    const float* qw;
    const float* ew;
    int normalize;
    int z_per_head;
};

// Workspace of the SMA forward: the key side r (.) dH of memories 0..M-2,
// [B][M-1][H][N][P] in the storage dtype.
size_t sma_workspace_bytes(const Shape& s);
hipError_t launch_sma(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                      const void* Cm, const void* mem, const void* z, const void* y_ssd, void* y,
                      float* lse, void* ws, hipStream_t st);

// Generic SMA forward (no workspace).
hipError_t launch_gsma(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                       const void* Cm, const void* mem, const void* z, const void* y_ssd, void* y,
                       float* lse, hipStream_t st);

// Workspace of the generic SMA backward: per (b, h, memory 0..M-2, token) the
// logit (then g p_j) and dy . V_j (then dl_j) with row stride Ls; Dy per
// (b, t, h); per-head token gradients [B][L][H][2N+P].
struct GenBwdWs {
    float* gp;
    float* dl;
    float* rdy;
    float* part;
    int64_t Ls;
    size_t bytes;  // total workspace
};
// Token and memory sides of the generic SMA backward (the caller finishes
// q, e, C and z gradients from part and rdy).
hipError_t launch_gsma_bwd(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                           const void* Cm, const void* mem, const void* z, const void* dy,
                           const GenBwdWs& w, float* dmem, hipStream_t st);

// Key side r (.) dH of memories 0..M-2 in the cache layout [B][M-1][H][N][P]
// (storage dtype), as the fp32 forward stages it; klo (optional, bf16 only,
// same layout) receives its rounding residual; rinv (optional,
// [B][M-1][H][N] float) receives 1 / r.
hipError_t launch_sma_keys(const Shape& s, const SmaArgs& a, const void* mem, void* kmem,
                           void* klo, float* rinv, hipStream_t st);

// SMA backward: key side, Qbar/Ebar, per-(head, memory, token) softmax
// scalars, per-head-block partial token gradients and R . dy.
size_t sma_bwd_workspace_bytes(const Shape& s);
hipError_t launch_sma_bwd(const Shape& s, const SmaArgs& a, const void* q, const void* e,
                          const void* Cm, const void* mem, const void* z, const float* lse,
                          const void* dy, float* dq, float* de, float* dC, float* dmem, float* dz,
                          void* ws, hipStream_t st);

// The block around the path (block.hip).
hipError_t launch_conv1d_silu(int dtype, int64_t B, int64_t L, int C, int64_t stride,
                              const void* in, const float* w, const float* bias,
                              const float* st_in, float* st_out, void* out, hipStream_t st);
hipError_t launch_dt_softplus(int dtype, int64_t rows, int H, const void* raw, int64_t stride,
                              const float* bias, float* dt, hipStream_t st);
hipError_t launch_gated_rmsnorm(int dtype, int64_t rows, int D, int group, const void* y,
                                const void* z, int64_t zstride, const float* w, float eps,
                                void* out, hipStream_t st);

// Backward of the block kernels (block.hip); workspaces hold per-block
// partial sums of the weight and bias gradients.
size_t conv1d_silu_bwd_workspace_bytes(int64_t B, int64_t L, int C);
hipError_t launch_conv1d_silu_bwd(int dtype, int64_t B, int64_t L, int C, int64_t stride,
                                  const void* in, const float* w, const float* bias,
                                  const float* st_in, const float* dout, float* din,
                                  int64_t dstride, float* dw, float* db, float* dst_in, void* ws,
                                  hipStream_t st);
size_t dt_softplus_bwd_workspace_bytes(int64_t rows, int H);
hipError_t launch_dt_softplus_bwd(int dtype, int64_t rows, int H, const void* raw, int64_t stride,
                                  const float* bias, const float* ddt, float* draw,
                                  int64_t dstride, float* dbias, void* ws, hipStream_t st);
size_t gated_rmsnorm_bwd_workspace_bytes(int64_t rows, int D);
hipError_t launch_gated_rmsnorm_bwd(int dtype, int64_t rows, int D, int group, const void* y,
                                    const void* z, int64_t zstride, const float* w, float eps,
                                    const float* dout, float* dy, float* dz, int64_t dzstride,
                                    float* dw, void* ws, hipStream_t st);

// Decode: per-split partial softmax statistics [B][H][nsplit][P+2] and the
// SSM readout y_ssd [B][H][P] (float).
constexpr int kDecodeMinMemPerSplit = 8;  // smallest split size the workspace allows
size_t decode_workspace_bytes(const Shape& s);
// pos_rows (device, [B]) == nullptr: every row at `pos`; otherwise row b at
// pos_rows[b], rows outside [0, pos] skipped, the grid sized for `pos`.
hipError_t launch_decode(const Shape& s, const SmaArgs& a, int64_t pos, const int64_t* pos_rows,
                         const void* x, const float* dt, const float* A, const void* Bm,
                         const void* Cm, const void* q, const void* e, const void* z,
                         float* h_state, float* chunk_acc, void* mem, void* y, void* ws,
                         hipStream_t st);
// The allocation-free decode step: the same kernels with the library's fixed
// device scratch (DART_DECODE_NOALLOC_SCRATCH_BYTES per device) as the
// workspace, laid out for this step's own split count.
size_t decode_noalloc_scratch_bytes(const Shape& s, int64_t pos);
hipError_t launch_decode_noalloc(const Shape& s, const SmaArgs& a, int64_t pos, const void* x,
                                 const float* dt, const float* A, const void* Bm, const void* Cm,
                                 const void* q, const void* e, const void* z, float* h_state,
                                 float* chunk_acc, void* mem, void* y, hipStream_t st);
hipError_t launch_decode_handoff(const Shape& s, const void* mem, const float* h_last,
                                 const int64_t* lengths, float* h_state, float* chunk_acc,
                                 hipStream_t st);

// Optional per-kernel timing (see dart_profile_* in dart.h).  Launchers
// bracket each kernel launch with prof_begin/prof_end; both are no-ops unless
// profiling is enabled.
void prof_begin(const char* kernel, hipStream_t st);
void prof_end(hipStream_t st);

inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }
// Compute units of the current device (queried once; 256 if the query fails).
int device_cu_count();
// Heads per block of the SMA kernels (forward and backward token kernels) for
// token blocks of tpb tokens: the power-of-2 divisor of H/G, at most hmax (the
// chooser's cap; the kernels take up to 8), with the least estimated makespan;
// no_first_chunk when the first chunk's blocks are not launched.
int sma_block_heads(int64_t B, int H, int G, int64_t L, int S, int tpb, int hmax,
                    bool no_first_chunk);
inline size_t elem_bytes(int dtype) { return dtype == 1 ? 2 : 4; }

}  // namespace dart
