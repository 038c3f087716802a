/*
 * dart.h -- C ABI of the DART hot-path library (libdart.so) for AMD Instinct
 * MI355X (gfx950).
 *
 * DART ("Decoded Attention over Recurrent sTates", arXiv 2608.02032) augments
 * the Mamba-2 chunked SSD scan: the scan keeps each chunk's state
 * contribution dH_[c] (a "chunk state memory", N x P per head), and
 * state-memory attention (SMA) lets every token attend over the memories of
 * strictly earlier chunks, decoding a token-conditioned key K = r (.) (dH E)
 * and value V = C dH from each memory, before a SiLU-gated residual adds the
 * readout to the SSM output.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensor pointers are DEVICE pointers to contiguous row-major arrays in the
 *    tensor order of the paper's App. B.2 (Table 7).  Symbols:
 *      B = batch, L = sequence length, H = heads, G = projection groups
 *      (G divides H; head h uses group h*G/H), P = head dim, N = state size,
 *      S = chunk size, M = ceil(L/S) chunks, Mcap = memory capacity >= M.
 *  - "storage dtype" (dims.dtype) is the element type of x, Bm, Cm, q, e, z,
 *    y_ssd, y and the memories: DART_FP32 (float) or DART_BF16 (bfloat16).
 *    dt, A, lse, h0, h_last, h_state and chunk_acc are always float.  All
 *    arithmetic accumulates in float.
 *  - Ownership: the caller allocates and owns every buffer, including the
 *    workspace.  The library allocates no memory, keeps no state between
 *    calls and is thread-safe; work is enqueued on `stream` (a hipStream_t;
 *    NULL = the null stream) and runs asynchronously.
 *  - Errors: every argument check runs on the host before any launch.  A
 *    failing check returns DART_ERR_INVALID_ARG (malformed arguments) or
 *    DART_ERR_UNSUPPORTED (well-formed shapes the library has no kernel for)
 *    and enqueues nothing; a failed launch returns DART_ERR_HIP.
 *    dart_last_error() gives a message for the last non-OK status of the
 *    calling thread.  Numeric contracts (dt > 0, A < 0) are the caller's.
 *  - Supported shapes: P = 64; N in {16, 32, 64, 128}; 1 <= S <= 4096; any
 *    L >= 1 (a partial last chunk is allowed); any B, H <= 65535 with
 *    H % G == 0.  N in {32, 64, 128} with S in {64, 128, 256} run the tuned
 *    MFMA kernels; every other shape runs generic fp32 kernels (the paper
 *    trains at S = 16, N in {16, 64} and evaluates at S = 32 and 64).
 *  - Tuning variables (results do not depend on them beyond floating-point
 *    summation order): DART_SMA_HEADS_PER_BLOCK in {1, 2, 4, 8} forces the
 *    number of heads one SMA workgroup serves (forward and backward; used
 *    when it divides H/G; read at every call, so it must not change between
 *    a workspace query and the call it sizes); DART_DECODE_MPS in
 *    {8, 16, 32, 64, 128} forces the memories per decode split (read once).
 *    Unset, both are chosen per shape.
 */
#ifndef DART_H
#define DART_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DART_OK = 0,
    DART_ERR_INVALID_ARG = 1,
    DART_ERR_UNSUPPORTED = 2,
    DART_ERR_HIP = 3
} dart_status;

typedef enum { DART_FP32 = 0, DART_BF16 = 1 } dart_dtype;

/* Problem dimensions (App. B.2 Table 7 symbols). */
typedef struct {
    int64_t batch;        /* B  >= 1 */
    int64_t seqlen;       /* L  >= 1 (ignored by the decode entry points) */
    int32_t nheads;       /* H  >= 1 */
    int32_t ngroups;      /* G  >= 1, H % G == 0 (the paper uses G = 1) */
    int32_t headdim;      /* P */
    int32_t dstate;       /* N */
    int32_t chunk;        /* S */
    int32_t dtype;        /* dart_dtype: storage dtype */
    int64_t mem_capacity; /* Mcap: slots in the memory array; 0 means ceil(L/S) */
} dart_dims;

/* State-memory attention options (Sec. 3 and App. B.1). */
typedef struct {
    float eps;              /* RMS epsilon for RMSNorm(Q), RMSNorm(E) and the memory
                               row inverse-RMS r; the paper leaves it open; > 0
                               required when normalize = 1 (1e-6 is the default of
                               the Python binding) */
    const float* q_norm_w;  /* device [N] RMSNorm weight of Q, or NULL for ones;
                               unused when normalize = 0 */
    const float* e_norm_w;  /* device [P] RMSNorm weight of E, or NULL for ones;
                               unused when normalize = 0 */
    int32_t normalize;      /* 1: normalised score branch of App. B.1;
                               0: Alg. 1 as printed (raw Q, E and r = 1) */
    int32_t z_per_head;     /* 1: z is [B][L][H] (one gate per head);
                               0: z is [B][L] (one scalar gate per token) */
} dart_sma_opts;

/* Bytes of workspace dart_ssd_chunk_scan needs for `dims`. */
size_t dart_scan_workspace_bytes(const dart_dims* dims);

/*
 * Mamba-2 chunked SSD scan that retains the chunk state memories.
 * Sec. 2 (SSD recurrence), Sec. 3 (chunk state memory dH_[c]) and App. A
 * (chunk-state, inter-chunk state passing, intra/inter-chunk outputs).  With
 * a_t = exp(dt_t * A_h) it computes, exactly up to rounding, the recurrence
 *     H_t = a_t H_{t-1} + dt_t B_t^T x_t,   y_ssd_t = C_t H_t,
 * starting from h0 (zero if NULL), and every chunk's contribution
 *     dH_[c] = sum_{s in chunk c} (prod_{k=s+1}^{e(c)} a_k) dt_s B_s^T x_s.
 *
 *   x      [B][L][H][P]     storage dtype, in
 *   dt     [B][L][H]        float, in (step sizes, already positive)
 *   A      [H]              float, in (negative decay rates)
 *   Bm, Cm [B][L][G][N]     storage dtype, in
 *   h0     [B][H][N][P]     float, in, or NULL
 *   y_ssd  [B][L][H][P]     storage dtype, out
 *   mem    [B][Mcap][H][N][P] storage dtype, out: slots 0..M-1 written (the
 *                           last one holds a partial chunk when L % S != 0),
 *                           slots >= M untouched.  Same layout as the decode
 *                           cache, so a prefill writes straight into it.
 *   h_last [B][H][N][P]     float, out, or NULL: H_{L-1}
 *   workspace               device buffer of >= dart_scan_workspace_bytes()
 */
dart_status dart_ssd_chunk_scan(const dart_dims* dims, const void* x, const float* dt,
                                const float* A, const void* Bm, const void* Cm, const float* h0,
                                void* y_ssd, void* mem, float* h_last, void* workspace,
                                size_t workspace_bytes, void* stream);

/* Bytes of workspace dart_ssd_bwd needs for `dims`: a forward scan's own
 * workspace and outputs, plus chunk adjoints, per-token decay pieces and
 * per-head-block dB / dC partials (all float). */
size_t dart_ssd_bwd_workspace_bytes(const dart_dims* dims);

/*
 * Backward of dart_ssd_chunk_scan (Sec. 2 recurrence, Sec. 3 / App. A chunk
 * memories): the gradients of
 *     sum dy . y_ssd + sum_c <dmem_c, dH_[c]> + <dh_last, H_{L-1}>
 * with respect to x, dt, A, Bm, Cm and h0, for the same inputs the forward
 * took.  The forward is recomputed inside (its chunk-entry states seed the
 * token sweeps), so nothing of a previous forward call is needed.  The
 * decay gradient is formed by the exact reverse-cumulative-sum identity
 *     d loss / d log a_t = sum_{s >= t} (y_s . dy_s - dx_s . x_s)
 *                          + <dh_last, H_{L-1}> + sum_{c' >= c(t)} <dmem_c', dH_[c']>,
 * then ddt_t = dx_t . x_t / dt_t + A_h (that), dA_h = sum_{b,t} dt_t (that).
 *
 *   x, dt, A, Bm, Cm, h0    as dart_ssd_chunk_scan (h0 may be NULL: zero)
 *   dy      [B][L][H][P]    storage dtype, in
 *   dmem    [B][Mcap][H][N][P] float, in, or NULL (slots 0..M-1 read)
 *   dh_last [B][H][N][P]    float, in, or NULL
 *   dx      [B][L][H][P]    float, out
 *   ddt     [B][L][H]       float, out
 *   dA      [H]             float, out (summed over the batch)
 *   dB, dC  [B][L][G][N]    float, out (summed over each group's heads)
 *   dh0     [B][H][N][P]    float, out, or NULL
 *   workspace               device buffer of >= dart_ssd_bwd_workspace_bytes()
 * Every output element is written (no accumulation into the caller's
 * buffers).  Deterministic: no atomics.
 */
dart_status dart_ssd_bwd(const dart_dims* dims, const void* x, const float* dt, const float* A,
                         const void* Bm, const void* Cm, const float* h0, const void* dy,
                         const float* dmem, const float* dh_last, float* dx, float* ddt, float* dA,
                         float* dB, float* dC, float* dh0, void* workspace, size_t workspace_bytes,
                         void* stream);

/* Bytes of workspace dart_sma_fwd needs for `dims`: the key side
 * r_j (.) dH_j of memories 0..M-2 in the cache layout (storage dtype); 0 when
 * M = 1 (workspace may then be NULL). */
size_t dart_sma_workspace_bytes(const dart_dims* dims);

/*
 * State-memory attention forward with the fused gated residual.
 * Sec. 3 ("State-Memory Attention", "Gated Residual Integration"), Alg. 1
 * (streaming over historical chunks with an online softmax; keys and values
 * decoded on chip) and App. B.1 (normalised score branch).  For token t of
 * chunk i = floor(t/S) and every memory j < i:
 *     Qb = RMSNorm(q_t) * q_norm_w,  Eb = RMSNorm(e_t) * e_norm_w,
 *     r_j[n] = (mean_p dH_j[n,p]^2 + eps)^-1/2,
 *     K = r_j (.) (dH_j Eb),  l_j = Qb . K / sqrt(N),  V_j = C_t dH_j,
 *     R_t = sum_j softmax_j(l)_j V_j,   LSE_t = log sum_j exp(l_j),
 *     y_t = y_ssd_t + SiLU(z_t) R_t.
 * Tokens of the first chunk have no history: R_t = 0, LSE_t = -inf and
 * y_t = y_ssd_t exactly.  r is computed from the memory values as stored.
 *
 *   q      [B][L][G][N]     storage dtype, in
 *   e      [B][L][G][P]     storage dtype, in
 *   Cm     [B][L][G][N]     storage dtype, in (the SSM read vector, shared)
 *   mem    [B][Mcap][H][N][P] storage dtype, in (slots 0..M-2 are read)
 *   z      [B][L][H] or [B][L] (opts->z_per_head) storage dtype, in: gate
 *                           pre-activation
 *   y_ssd  [B][L][H][P]     storage dtype, in
 *   y      [B][L][H][P]     storage dtype, out; may alias y_ssd exactly
 *   lse    [B][L][H]        float, out, or NULL
 *   workspace               device buffer of >= dart_sma_workspace_bytes()
 */
dart_status dart_sma_fwd(const dart_dims* dims, const dart_sma_opts* opts, const void* q,
                         const void* e, const void* Cm, const void* mem, const void* z,
                         const void* y_ssd, void* y, float* lse, void* workspace,
                         size_t workspace_bytes, void* stream);

/* Bytes of workspace dart_sma_bwd needs for `dims`: the key side of
 * memories 0..M-2 (as dart_sma_workspace_bytes for fp32), the normalised
 * query and E rows, two floats per (b, head, memory 0..M-2, token), the
 * per-head-block partial token gradients and one float per (b, token, head). */
size_t dart_sma_bwd_workspace_bytes(const dart_dims* dims);

/*
 * Backward of dart_sma_fwd for the loss sum_t dy_t . y_t (App. C: the scores
 * are recomputed and the softmax weights recovered as exp(l_j - LSE_t) from
 * the forward's log-sum-exp; the chain rule through the definitions of Sec. 3
 * and App. B.1, with the RMSNorm weights held constant).  With
 * g = SiLU(z_t), p_j the softmax weights and Dy = R_t . dy_t:
 *     dl_j = g p_j (dy_t . V_j - Dy),      dz_t = SiLU'(z_t) Dy,
 *     dC_t = sum_j g p_j dH_j dy_t,        dQbar = sum_j dl_j K_j / sqrt(N),
 *     dEbar = sum_j dH_j^T (r_j (.) Qbar) dl_j / sqrt(N),
 *     ddH_j = sum_t [g p_j C_t^T dy_t + r_j (.) (dl_j Qbar^T Ebar) / sqrt(N)]
 *             - (r_j^3 / P) (.) rowsum(dH_j (.) that second sum) (.) dH_j,
 * then dq and de through RMSNorm.  This is the attention branch only: the
 * gradient of y with respect to y_ssd is dy itself, and the scan's own
 * backward is not part of this call.
 *
 *   q, e, Cm, mem, z  as in dart_sma_fwd (storage dtype, in)
 *   lse    [B][L][H]        float, in: the forward's log-sum-exp
 *   dy     [B][L][H][P]     storage dtype, in: gradient of y
 *   dq     [B][L][G][N]     float, out (summed over the heads of a group)
 *   de     [B][L][G][P]     float, out (summed over the heads of a group)
 *   dC     [B][L][G][N]     float, out: the attention branch's part of the
 *                           gradient of C (summed over the heads of a group)
 *   dmem   [B][Mcap][H][N][P] float, out: every slot written (slots M-1 and
 *                           above, which no token attends, are zero)
 *   dz     like z           float, out
 *   workspace               device buffer of >= dart_sma_bwd_workspace_bytes()
 * Tokens of the first chunk get zero q, e, C and z gradients.  Deterministic:
 * no atomics, every sum has a fixed order.
 */
dart_status dart_sma_bwd(const dart_dims* dims, const dart_sma_opts* opts, const void* q,
                         const void* e, const void* Cm, const void* mem, const void* z,
                         const float* lse, const void* dy, float* dq, float* de, float* dC,
                         float* dmem, float* dz, void* workspace, size_t workspace_bytes,
                         void* stream);

/*
 * The steps either side of the path in the DART (Mamba-2) block.  The paper
 * fixes the convolution width (4) and RMSNorm (App. D.2, with Table 8); the
 * conventions below are those of the Mamba-2 block it builds on.  All three
 * are stream-ordered elementwise or row-local kernels; none allocates.
 *
 * dart_conv1d_silu: causal depthwise convolution of width 4 over the token
 * axis with bias and SiLU, on the x, B and C channels of the input
 * projection:  out[b][t][c] = SiLU(bias[c] + sum_{k=0..3} w[c][k] in[b][t-3+k][c]),
 * where in[b][s][c] for s < 0 is state_in[b][c][3+s] (zero when state_in is
 * NULL).  state_out (optional) receives the last three inputs of each
 * channel, oldest first: the decode cache of the convolution, so a call
 * over tokens 0..L-1 followed by one over L.. with that state equals one call
 * over both (a decode step is seqlen = 1).
 *   in         [B][L][row_stride] storage dtype, channel c at element c of
 *              the row (pass a pointer to the first x channel of the
 *              projection output)
 *   weight     [C][4] float (weight[c][3] multiplies the current token)
 *   bias       [C] float, or NULL
 *   state_in   [B][C][3] float, or NULL;  state_out [B][C][3] float, or NULL
 *              (state_out may equal state_in when seqlen <= 32)
 *   out        [B][L][C] storage dtype
 */
dart_status dart_conv1d_silu(int64_t batch, int64_t seqlen, int32_t channels, int64_t row_stride,
                             int32_t dtype, const void* in, const float* weight, const float* bias,
                             const float* state_in, float* state_out, void* out, void* stream);

/*
 * Step sizes from the projection: dt[r][h] = softplus(raw[r][h] + bias[h])
 * = log(1 + exp(.)), in float (the scan takes dt already positive).
 *   raw  [rows][row_stride] storage dtype (head h at element h of the row)
 *   bias [H] float, or NULL;  dt [rows][H] float
 */
dart_status dart_dt_softplus(int64_t rows, int32_t nheads, int64_t row_stride, int32_t dtype,
                             const void* raw, const float* bias, float* dt, void* stream);

/*
 * Gated RMSNorm ahead of the output projection: with u = y (.) SiLU(z),
 *   out = u / sqrt(mean over its group of u^2 + eps) (.) weight,
 * over consecutive groups of `group` channels of each row (group = dim for
 * one group).
 *   y, out [rows][dim] storage dtype;  z [rows][z_row_stride] storage dtype
 *   (the gate channels of the projection output);  weight [dim] float or NULL
 * Requirements: group divides dim, group and z_row_stride multiples of 8,
 * y, z, out and weight 16-byte aligned, eps > 0.
 */
dart_status dart_gated_rmsnorm(int64_t rows, int32_t dim, int32_t group, int32_t dtype,
                               const void* y, const void* z, int64_t z_row_stride,
                               const float* weight, float eps, void* out, void* stream);

/*
 * Backward of the three block kernels above, for a loss whose gradient with
 * respect to the kernel's output is `dout` (float).  Gradients are float and
 * overwrite their outputs; the sums over tokens or rows (weights, biases) are
 * formed from per-block partials in the workspace in a fixed order
 * (deterministic).  The forward inputs are passed again (nothing of the
 * forward call is kept).
 *
 * dart_conv1d_silu_bwd: with u = bias + sum_k w_k in[t-3+k] (the forward's
 * pre-activation) and du = dout SiLU'(u):
 *   din[t] = sum_k w_k du[t+3-k]   [B][L][din_row_stride] (channel c at c)
 *   dweight[c][k] = sum_{b,t} du in[t-3+k]   [C][4];   dbias [C] or NULL
 *   dstate_in [B][C][3] or NULL: the gradient of the carried state
 *   (in[-3..-1]; zero-state inputs get it too)
 *   in, weight, bias, state_in, row_stride, dtype as in dart_conv1d_silu.
 */
size_t dart_conv1d_silu_bwd_workspace_bytes(int64_t batch, int64_t seqlen, int32_t channels);
dart_status dart_conv1d_silu_bwd(int64_t batch, int64_t seqlen, int32_t channels,
                                 int64_t row_stride, int32_t dtype, const void* in,
                                 const float* weight, const float* bias, const float* state_in,
                                 const float* dout, float* din, int64_t din_row_stride,
                                 float* dweight, float* dbias, float* dstate_in, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* dart_dt_softplus_bwd: draw = ddt sigmoid(raw + bias) [rows][draw_row_stride]
 * (head h at h), dbias [H] = sum over rows, or NULL.  ddt [rows][H] float. */
size_t dart_dt_softplus_bwd_workspace_bytes(int64_t rows, int32_t nheads);
dart_status dart_dt_softplus_bwd(int64_t rows, int32_t nheads, int64_t row_stride, int32_t dtype,
                                 const void* raw, const float* bias, const float* ddt, float* draw,
                                 int64_t draw_row_stride, float* dbias, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* dart_gated_rmsnorm_bwd: with u = y SiLU(z), inv = (mean over the group of
 * u^2 + eps)^-1/2 and g = dout (.) weight:
 *   du = inv g - u inv^3 (g . u) / group,  dy = du SiLU(z)  [rows][dim],
 *   dz = du y SiLU'(z)  [rows][dz_row_stride],
 *   dweight [dim] = sum over rows of dout u inv, or NULL.
 * Groups of at most 2048 channels; y, z, dout, dy, dz 32-byte aligned; row
 * strides multiples of 8. */
size_t dart_gated_rmsnorm_bwd_workspace_bytes(int64_t rows, int32_t dim);
dart_status dart_gated_rmsnorm_bwd(int64_t rows, int32_t dim, int32_t group, int32_t dtype,
                                   const void* y, const void* z, int64_t z_row_stride,
                                   const float* weight, float eps, const float* dout, float* dy,
                                   float* dz, int64_t dz_row_stride, float* dweight,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace dart_decode_step needs (dims->seqlen is ignored; the
 * worst case over positions that fit dims->mem_capacity is returned). */
size_t dart_decode_workspace_bytes(const dart_dims* dims);

/*
 * One autoregressive decode step at 0-based position `pos` (host value, the
 * same for every sequence), over the cached chunk memories.  The paper gives
 * no algorithm for it (Sec. 4 "Inference Cache" names the caches); the order
 * is the one that reproduces the forward pass token by token:
 *   1. if pos % S == 0: chunk_acc = 0 (a new chunk starts);
 *   2. a = exp(dt A_h); h_state = a h_state + dt B^T x; chunk_acc likewise;
 *   3. y_ssd = C h_state;
 *   4. SMA (as in dart_sma_fwd) over memories 0 .. m-1, m = floor(pos/S);
 *   5. y = y_ssd + SiLU(z) R;
 *   6. if pos % S == S-1: mem_cache[m] = chunk_acc (rounded to storage dtype).
 * After step 6 chunk_acc equals dH_[m] and h_state equals H_pos.
 *
 *   x       [B][H][P]       storage dtype, in
 *   dt      [B][H]          float, in
 *   A       [H]             float, in
 *   Bm, Cm, q [B][G][N]     storage dtype, in
 *   e       [B][G][P]       storage dtype, in
 *   z       [B][H] or [B]   storage dtype, in
 *   h_state [B][H][N][P]    float, in/out
 *   chunk_acc [B][H][N][P]  float, in/out
 *   mem_cache [B][Mcap][H][N][P] storage dtype, in/out (slot m written on
 *                           step 6 only); Mcap = dims->mem_capacity (> 0)
 *   y       [B][H][P]       storage dtype, out
 * Errors: DART_ERR_INVALID_ARG if pos < 0, if m > Mcap, or if the step would
 * append (pos % S == S-1) with m >= Mcap.
 */
dart_status dart_decode_step(const dart_dims* dims, const dart_sma_opts* opts, int64_t pos,
                             const void* x, const float* dt, const float* A, const void* Bm,
                             const void* Cm, const void* q, const void* e, const void* z,
                             float* h_state, float* chunk_acc, void* mem_cache, void* y,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * dart_decode_step for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same step, arguments and errors as dart_decode_step, with
 * no workspace argument.  Its partial softmax statistics and SSM readout go
 * to a fixed scratch array the library holds on each device it runs on, of
 * DART_DECODE_NOALLOC_SCRATCH_BYTES (16 MiB), kept until the process ends;
 * the step needs B * H * (nsplit * (P + 2) + P) * 4 bytes of it, nsplit the
 * number of memory splits of the step (at most ceil(m / 8)), e.g. 1.6 MB for
 * B = 64, H = 32 and 256 cached memories.  A step that needs more returns
 * DART_ERR_UNSUPPORTED before any launch.  The scratch is that of the device
 * current on the calling thread, which must be the device of `stream` and of
 * every buffer.  Every call on a device shares its scratch: calls that
 * overlap in time on one device (several streams, or threads without
 * ordering) race, so issue them in one stream order.  Nothing in the scratch
 * needs clearing: every value a step reads was written by that step.  This
 * function allocates nothing.
 */
#define DART_DECODE_NOALLOC_SCRATCH_BYTES (16u << 20)
dart_status dart_decode_step_noalloc(const dart_dims* dims, const dart_sma_opts* opts, int64_t pos,
                                     const void* x, const float* dt, const float* A,
                                     const void* Bm, const void* Cm, const void* q, const void* e,
                                     const void* z, float* h_state, float* chunk_acc,
                                     void* mem_cache, void* y, void* stream);

/*
 * The decode step for a ragged batch: row b of the batch is at its own
 * 0-based position pos[b] and runs steps 1-6 of dart_decode_step at that
 * position (reset, append and the number m_b = floor(pos[b]/S) of memories it
 * attends all follow pos[b]).  Sec. 4 ("Inference Cache") keeps one cache per
 * sequence; a batch of sequences of different lengths shares these buffers.
 *
 *   pos      [B] int64, device, in: the rows' positions
 *   pos_max  host: an upper bound of pos[] that sizes the launch; rows with
 *            pos[b] < 0 or pos[b] > pos_max take no part in the step (their
 *            state, cache and y are left as they are)
 *   other arguments, layouts and the workspace as in dart_decode_step.
 * Errors: DART_ERR_INVALID_ARG if pos_max < 0 or pos_max >= S * Mcap (some
 * row could then need a memory slot the cache does not have).
 */
dart_status dart_decode_step_ragged(const dart_dims* dims, const dart_sma_opts* opts,
                                    const int64_t* pos, int64_t pos_max, const void* x,
                                    const float* dt, const float* A, const void* Bm,
                                    const void* Cm, const void* q, const void* e, const void* z,
                                    float* h_state, float* chunk_acc, void* mem_cache, void* y,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * Prefill -> decode handoff.  After dart_ssd_chunk_scan over a batch padded to
 * a common length with dt = 0 on each row's padding (decay 1 and no input, so
 * the state, h_last and every memory equal those of the row's own prefix),
 * the decode state of row b for its next position L_b = lengths[b]:
 *   h_state[b]   = h_last[b];
 *   chunk_acc[b] = mem[b][floor(L_b/S)] (the running contribution of the
 *                  partial chunk, as stored) if L_b % S != 0, else 0.
 * mem is the scan's memory output written with capacity dims->mem_capacity,
 * which then serves as the decode cache as is (slots below floor(L_b/S) hold
 * the row's completed chunks).  Rows with lengths[b] < 0 are left untouched.
 * The caller keeps ceil(L_b/S) <= mem_capacity.
 *
 *   lengths  [B] int64, device, in
 *   mem      [B][Mcap][H][N][P] storage dtype, in
 *   h_last   [B][H][N][P] float, in
 *   h_state, chunk_acc [B][H][N][P] float, out
 */
dart_status dart_decode_handoff(const dart_dims* dims, const int64_t* lengths, const void* mem,
                                const float* h_last, float* h_state, float* chunk_acc,
                                void* stream);

/*
 * Element count of the length-dependent decode cache for a context of
 * `context` tokens: B * ceil(context/S) * H * N * P chunk-memory elements
 * (Sec. 4 "Inference Cache": O(M N P) per head).  The matched token-attention
 * KV cache is B * H * 2 * context * P elements, so for context % S == 0 the
 * ratio is N / (2 S).  Returns 0 for malformed dims.
 */
int64_t dart_decode_cache_elems(const dart_dims* dims, int64_t context);

const char* dart_status_string(dart_status status);
const char* dart_last_error(void);

/*
 * Optional kernel timing (a tracing aid, off by default).  While enabled,
 * every kernel the library launches -- or, after dart_profile_filter(name),
 * only the kernel of that name (e.g. "k_sma") -- is bracketed by two HIP
 * events recorded on the stream it is launched on.  dart_profile_flush()
 * waits for the pending events and adds each kernel's elapsed time to a
 * per-kernel total; the totals are read by index (0 .. dart_profile_count()-1)
 * and cleared, with the filter, by dart_profile_reset().  Events are created
 * on first use and kept for reuse until dart_profile_reset(); this is the only
 * state the library keeps.  The totals are shared by all threads under one
 * lock and every launching thread pairs its own events, so the functions may
 * be called from several threads; a reset while another thread launches
 * drops that thread's open interval.  dart_profile_flush() returns
 * DART_ERR_HIP if an event query fails.
 */
dart_status dart_profile_enable(int enable);
dart_status dart_profile_filter(const char* kernel);  /* NULL or "": every kernel */
dart_status dart_profile_flush(void);
int dart_profile_count(void);
const char* dart_profile_name(int index);     /* kernel name, or NULL */
double dart_profile_total_ms(int index);      /* summed elapsed ms */
int64_t dart_profile_launches(int index);     /* number of timed launches */
void dart_profile_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* DART_H */
