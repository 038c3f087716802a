// dart_api.cpp -- the C ABI of libdart.so (declared in include/dart.h):
// argument validation on the host, workspace sizing, dispatch to the kernel
// launchers, status codes and a per-thread error message.  Nothing here
// allocates device memory or keeps state between calls.
#include "dart.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdint>
#include <cstring>

#include "dart_internal.hpp"

namespace {

thread_local char g_err[512] = "";

dart_status fail(dart_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

dart_status ok() {
    g_err[0] = '\0';
    return DART_OK;
}

// Checks shared by every entry point; fills `s` on success.
dart_status make_shape(const dart_dims* d, bool need_seqlen, dart::Shape& s) {
    if (!d) return fail(DART_ERR_INVALID_ARG, "dims is NULL");
    if (d->batch < 1) return fail(DART_ERR_INVALID_ARG, "batch must be >= 1 (got %lld)", (long long)d->batch);
    if (need_seqlen && d->seqlen < 1)
        return fail(DART_ERR_INVALID_ARG, "seqlen must be >= 1 (got %lld)", (long long)d->seqlen);
    if (d->nheads < 1 || d->ngroups < 1)
        return fail(DART_ERR_INVALID_ARG, "nheads and ngroups must be >= 1");
    if (d->nheads % d->ngroups != 0)
        return fail(DART_ERR_INVALID_ARG, "nheads (%d) must be a multiple of ngroups (%d)", d->nheads, d->ngroups);
    if (d->headdim < 1 || d->dstate < 1 || d->chunk < 1)
        return fail(DART_ERR_INVALID_ARG, "headdim, dstate and chunk must be >= 1");
    if (d->dtype != DART_FP32 && d->dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", d->dtype);
    if (d->mem_capacity < 0) return fail(DART_ERR_INVALID_ARG, "mem_capacity must be >= 0");
    if (d->headdim != 64)
        return fail(DART_ERR_UNSUPPORTED, "headdim %d not supported (the library has kernels for 64)", d->headdim);
    if (d->dstate != 16 && d->dstate != 32 && d->dstate != 64 && d->dstate != 128)
        return fail(DART_ERR_UNSUPPORTED, "dstate %d not supported (16, 32, 64 or 128)", d->dstate);
    if (d->chunk > 4096)
        return fail(DART_ERR_UNSUPPORTED, "chunk %d not supported (at most 4096)", d->chunk);
    if (d->batch > 65535 || d->nheads > 65535)
        return fail(DART_ERR_UNSUPPORTED, "batch and nheads must be <= 65535");
    s.B = d->batch;
    s.L = need_seqlen ? d->seqlen : 0;
    s.H = d->nheads;
    s.G = d->ngroups;
    s.P = d->headdim;
    s.N = d->dstate;
    s.S = d->chunk;
    s.M = need_seqlen ? (s.L + s.S - 1) / s.S : 0;
    s.Mcap = d->mem_capacity ? d->mem_capacity : s.M;
    s.dtype = d->dtype;
    if (need_seqlen && s.Mcap < s.M)
        return fail(DART_ERR_INVALID_ARG, "mem_capacity %lld < ceil(L/S) = %lld", (long long)s.Mcap,
                    (long long)s.M);
    if (need_seqlen && s.M > 2147483647LL) return fail(DART_ERR_UNSUPPORTED, "too many chunks");
    return DART_OK;
}

dart_status check_opts(const dart_sma_opts* o) {
    if (!o) return fail(DART_ERR_INVALID_ARG, "opts is NULL");
    if (o->normalize != 0 && o->normalize != 1) return fail(DART_ERR_INVALID_ARG, "normalize must be 0 or 1");
    if (o->z_per_head != 0 && o->z_per_head != 1) return fail(DART_ERR_INVALID_ARG, "z_per_head must be 0 or 1");
    if (o->normalize && !(o->eps > 0.0f)) return fail(DART_ERR_INVALID_ARG, "eps must be > 0 when normalize = 1");
    if (!(o->eps >= 0.0f)) return fail(DART_ERR_INVALID_ARG, "eps must be >= 0");
    return DART_OK;
}

// The norm weights belong to RMSNorm: without normalisation they are unused.
dart::SmaArgs sma_args(const dart_sma_opts* o) {
    return dart::SmaArgs{o->eps, o->normalize ? o->q_norm_w : nullptr,
                         o->normalize ? o->e_norm_w : nullptr, o->normalize, o->z_per_head};
}

dart_status hip_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(DART_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

#define REQUIRE_PTR(p) \
    if (!(p)) return fail(DART_ERR_INVALID_ARG, "required pointer '%s' is NULL", #p)

}  // namespace

extern "C" {

size_t dart_scan_workspace_bytes(const dart_dims* dims) {
    dart::Shape s;
    if (make_shape(dims, true, s) != DART_OK) return 0;
    return dart::scan_workspace_bytes(s);
}

dart_status dart_ssd_chunk_scan(const dart_dims* dims, const void* x, const float* dt,
                                const float* A, const void* Bm, const void* Cm, const float* h0,
                                void* y_ssd, void* mem, float* h_last, void* workspace,
                                size_t workspace_bytes, void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, true, s);
    if (st != DART_OK) return st;
    REQUIRE_PTR(x);
    REQUIRE_PTR(dt);
    REQUIRE_PTR(A);
    REQUIRE_PTR(Bm);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(y_ssd);
    REQUIRE_PTR(mem);
    REQUIRE_PTR(workspace);
    const size_t need = dart::scan_workspace_bytes(s);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return hip_status(dart::launch_scan(s, x, dt, A, Bm, Cm, h0, y_ssd, mem, h_last, workspace,
                                        (hipStream_t)stream),
                      "dart_ssd_chunk_scan launch");
}

size_t dart_ssd_bwd_workspace_bytes(const dart_dims* dims) {
    dart::Shape s;
    if (make_shape(dims, true, s) != DART_OK) return 0;
    return dart::ssd_bwd_workspace_bytes(s);
}

dart_status dart_ssd_bwd(const dart_dims* dims, const void* x, const float* dt, const float* A,
                         const void* Bm, const void* Cm, const float* h0, const void* dy,
                         const float* dmem, const float* dh_last, float* dx, float* ddt, float* dA,
                         float* dB, float* dC, float* dh0, void* workspace, size_t workspace_bytes,
                         void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, true, s);
    if (st != DART_OK) return st;
    REQUIRE_PTR(x);
    REQUIRE_PTR(dt);
    REQUIRE_PTR(A);
    REQUIRE_PTR(Bm);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(dy);
    REQUIRE_PTR(dx);
    REQUIRE_PTR(ddt);
    REQUIRE_PTR(dA);
    REQUIRE_PTR(dB);
    REQUIRE_PTR(dC);
    REQUIRE_PTR(workspace);
    const size_t need = dart::ssd_bwd_workspace_bytes(s);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return hip_status(dart::launch_ssd_bwd(s, x, dt, A, Bm, Cm, h0, dy, dmem, dh_last, dx, ddt, dA,
                                           dB, dC, dh0, workspace, (hipStream_t)stream),
                      "dart_ssd_bwd launch");
}

size_t dart_sma_workspace_bytes(const dart_dims* dims) {
    dart::Shape s;
    if (make_shape(dims, true, s) != DART_OK) return 0;
    return dart::sma_workspace_bytes(s);
}

dart_status dart_sma_fwd(const dart_dims* dims, const dart_sma_opts* opts, const void* q,
                         const void* e, const void* Cm, const void* mem, const void* z,
                         const void* y_ssd, void* y, float* lse, void* workspace,
                         size_t workspace_bytes, void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, true, s);
    if (st != DART_OK) return st;
    st = check_opts(opts);
    if (st != DART_OK) return st;
    REQUIRE_PTR(q);
    REQUIRE_PTR(e);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(mem);
    REQUIRE_PTR(z);
    REQUIRE_PTR(y_ssd);
    REQUIRE_PTR(y);
    const size_t need = dart::sma_workspace_bytes(s);
    if (need > 0 && !workspace) return fail(DART_ERR_INVALID_ARG, "required pointer 'workspace' is NULL");
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    if (y != y_ssd) {
        // partial overlap between y and y_ssd is not allowed (exact aliasing is)
        const size_t bytes = (size_t)s.B * s.L * s.H * s.P * dart::elem_bytes(s.dtype);
        const char* a0 = (const char*)y;
        const char* b0 = (const char*)y_ssd;
        if (a0 < b0 + bytes && b0 < a0 + bytes)
            return fail(DART_ERR_INVALID_ARG, "y partially overlaps y_ssd (only exact aliasing is allowed)");
    }
    const dart::SmaArgs a = sma_args(opts);
    return hip_status(dart::launch_sma(s, a, q, e, Cm, mem, z, y_ssd, y, lse, workspace,
                                       (hipStream_t)stream),
                      "dart_sma_fwd launch");
}

size_t dart_sma_bwd_workspace_bytes(const dart_dims* dims) {
    dart::Shape s;
    if (make_shape(dims, true, s) != DART_OK) return 0;
    return dart::sma_bwd_workspace_bytes(s);
}

dart_status dart_sma_bwd(const dart_dims* dims, const dart_sma_opts* opts, const void* q,
                         const void* e, const void* Cm, const void* mem, const void* z,
                         const float* lse, const void* dy, float* dq, float* de, float* dC,
                         float* dmem, float* dz, void* workspace, size_t workspace_bytes,
                         void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, true, s);
    if (st != DART_OK) return st;
    st = check_opts(opts);
    if (st != DART_OK) return st;
    REQUIRE_PTR(q);
    REQUIRE_PTR(e);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(mem);
    REQUIRE_PTR(z);
    REQUIRE_PTR(lse);
    REQUIRE_PTR(dy);
    REQUIRE_PTR(dq);
    REQUIRE_PTR(de);
    REQUIRE_PTR(dC);
    REQUIRE_PTR(dmem);
    REQUIRE_PTR(dz);
    REQUIRE_PTR(workspace);
    const size_t need = dart::sma_bwd_workspace_bytes(s);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return hip_status(dart::launch_sma_bwd(s, sma_args(opts), q, e, Cm, mem, z, lse, dy, dq, de, dC,
                                           dmem, dz, workspace, (hipStream_t)stream),
                      "dart_sma_bwd launch");
}

dart_status dart_conv1d_silu(int64_t batch, int64_t seqlen, int32_t channels, int64_t row_stride,
                             int32_t dtype, const void* in, const float* weight, const float* bias,
                             const float* state_in, float* state_out, void* out, void* stream) {
    if (batch < 1 || seqlen < 1 || channels < 1)
        return fail(DART_ERR_INVALID_ARG, "batch, seqlen and channels must be >= 1");
    if (batch > 65535 || (seqlen + 31) / 32 > 65535)
        return fail(DART_ERR_UNSUPPORTED, "batch <= 65535 and seqlen <= 32 * 65535");
    if (row_stride < channels)
        return fail(DART_ERR_INVALID_ARG, "row_stride (%lld) < channels (%d)", (long long)row_stride, channels);
    if (dtype != DART_FP32 && dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", dtype);
    REQUIRE_PTR(in);
    REQUIRE_PTR(weight);
    REQUIRE_PTR(out);
    if (state_out && state_out == state_in && seqlen > 32)
        return fail(DART_ERR_INVALID_ARG, "state_out may alias state_in only for seqlen <= 32");
    return hip_status(dart::launch_conv1d_silu(dtype, batch, seqlen, channels, row_stride, in, weight,
                                               bias, state_in, state_out, out, (hipStream_t)stream),
                      "dart_conv1d_silu launch");
}

dart_status dart_dt_softplus(int64_t rows, int32_t nheads, int64_t row_stride, int32_t dtype,
                             const void* raw, const float* bias, float* dt, void* stream) {
    if (rows < 1 || nheads < 1) return fail(DART_ERR_INVALID_ARG, "rows and nheads must be >= 1");
    if (row_stride < nheads)
        return fail(DART_ERR_INVALID_ARG, "row_stride (%lld) < nheads (%d)", (long long)row_stride, nheads);
    if (dtype != DART_FP32 && dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", dtype);
    if ((rows * nheads + 255) / 256 > 2147483647LL) return fail(DART_ERR_UNSUPPORTED, "too many rows");
    REQUIRE_PTR(raw);
    REQUIRE_PTR(dt);
    return hip_status(dart::launch_dt_softplus(dtype, rows, nheads, raw, row_stride, bias, dt,
                                               (hipStream_t)stream),
                      "dart_dt_softplus launch");
}

dart_status dart_gated_rmsnorm(int64_t rows, int32_t dim, int32_t group, int32_t dtype,
                               const void* y, const void* z, int64_t z_row_stride,
                               const float* weight, float eps, void* out, void* stream) {
    if (rows < 1 || dim < 1 || group < 1) return fail(DART_ERR_INVALID_ARG, "rows, dim and group must be >= 1");
    if (dim % group != 0 || group % 8 != 0)
        return fail(DART_ERR_INVALID_ARG, "group must divide dim and be a multiple of 8 (dim %d, group %d)", dim, group);
    if (z_row_stride < dim || z_row_stride % 8 != 0)
        return fail(DART_ERR_INVALID_ARG, "z_row_stride must be >= dim and a multiple of 8");
    if (dtype != DART_FP32 && dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", dtype);
    if (!(eps > 0.0f)) return fail(DART_ERR_INVALID_ARG, "eps must be > 0");
    REQUIRE_PTR(y);
    REQUIRE_PTR(z);
    REQUIRE_PTR(out);
    if (((uintptr_t)y | (uintptr_t)z | (uintptr_t)out | (uintptr_t)weight) % 16 != 0)
        return fail(DART_ERR_INVALID_ARG, "y, z, out and weight must be 16-byte aligned");
    if ((rows * (dim / group) + 3) / 4 > 2147483647LL) return fail(DART_ERR_UNSUPPORTED, "too many rows");
    return hip_status(dart::launch_gated_rmsnorm(dtype, rows, dim, group, y, z, z_row_stride, weight,
                                                 eps, out, (hipStream_t)stream),
                      "dart_gated_rmsnorm launch");
}

size_t dart_conv1d_silu_bwd_workspace_bytes(int64_t batch, int64_t seqlen, int32_t channels) {
    if (batch < 1 || seqlen < 1 || channels < 1) return 0;
    return dart::conv1d_silu_bwd_workspace_bytes(batch, seqlen, channels);
}

dart_status dart_conv1d_silu_bwd(int64_t batch, int64_t seqlen, int32_t channels,
                                 int64_t row_stride, int32_t dtype, const void* in,
                                 const float* weight, const float* bias, const float* state_in,
                                 const float* dout, float* din, int64_t din_row_stride,
                                 float* dweight, float* dbias, float* dstate_in, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    if (batch < 1 || seqlen < 1 || channels < 1)
        return fail(DART_ERR_INVALID_ARG, "batch, seqlen and channels must be >= 1");
    if (batch > 65535 || (seqlen + 31) / 32 > 65535)
        return fail(DART_ERR_UNSUPPORTED, "batch <= 65535 and seqlen <= 32 * 65535");
    if (row_stride < channels || din_row_stride < channels)
        return fail(DART_ERR_INVALID_ARG, "row strides must be >= channels (%d)", channels);
    if (dtype != DART_FP32 && dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", dtype);
    REQUIRE_PTR(in);
    REQUIRE_PTR(weight);
    REQUIRE_PTR(dout);
    REQUIRE_PTR(din);
    REQUIRE_PTR(dweight);
    REQUIRE_PTR(workspace);
    const size_t need = dart::conv1d_silu_bwd_workspace_bytes(batch, seqlen, channels);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return hip_status(dart::launch_conv1d_silu_bwd(dtype, batch, seqlen, channels, row_stride, in,
                                                   weight, bias, state_in, dout, din,
                                                   din_row_stride, dweight, dbias, dstate_in,
                                                   workspace, (hipStream_t)stream),
                      "dart_conv1d_silu_bwd launch");
}

size_t dart_dt_softplus_bwd_workspace_bytes(int64_t rows, int32_t nheads) {
    if (rows < 1 || nheads < 1) return 0;
    return dart::dt_softplus_bwd_workspace_bytes(rows, nheads);
}

dart_status dart_dt_softplus_bwd(int64_t rows, int32_t nheads, int64_t row_stride, int32_t dtype,
                                 const void* raw, const float* bias, const float* ddt, float* draw,
                                 int64_t draw_row_stride, float* dbias, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    if (rows < 1 || nheads < 1) return fail(DART_ERR_INVALID_ARG, "rows and nheads must be >= 1");
    if (row_stride < nheads || draw_row_stride < nheads)
        return fail(DART_ERR_INVALID_ARG, "row strides must be >= nheads (%d)", nheads);
    if (dtype != DART_FP32 && dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", dtype);
    if ((rows + 255) / 256 > 65535) return fail(DART_ERR_UNSUPPORTED, "too many rows");
    REQUIRE_PTR(raw);
    REQUIRE_PTR(ddt);
    REQUIRE_PTR(draw);
    REQUIRE_PTR(workspace);
    const size_t need = dart::dt_softplus_bwd_workspace_bytes(rows, nheads);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    return hip_status(dart::launch_dt_softplus_bwd(dtype, rows, nheads, raw, row_stride, bias, ddt,
                                                   draw, draw_row_stride, dbias, workspace,
                                                   (hipStream_t)stream),
                      "dart_dt_softplus_bwd launch");
}

size_t dart_gated_rmsnorm_bwd_workspace_bytes(int64_t rows, int32_t dim) {
    if (rows < 1 || dim < 1) return 0;
    return dart::gated_rmsnorm_bwd_workspace_bytes(rows, dim);
}

dart_status dart_gated_rmsnorm_bwd(int64_t rows, int32_t dim, int32_t group, int32_t dtype,
                                   const void* y, const void* z, int64_t z_row_stride,
                                   const float* weight, float eps, const float* dout, float* dy,
                                   float* dz, int64_t dz_row_stride, float* dweight,
                                   void* workspace, size_t workspace_bytes, void* stream) {
    if (rows < 1 || dim < 1 || group < 1) return fail(DART_ERR_INVALID_ARG, "rows, dim and group must be >= 1");
    if (dim % group != 0 || group % 8 != 0)
        return fail(DART_ERR_INVALID_ARG, "group must divide dim and be a multiple of 8 (dim %d, group %d)", dim, group);
    if (group > 2048) return fail(DART_ERR_UNSUPPORTED, "the backward supports groups of at most 2048 channels");
    if (z_row_stride < dim || z_row_stride % 8 != 0 || dz_row_stride < dim || dz_row_stride % 8 != 0)
        return fail(DART_ERR_INVALID_ARG, "z and dz row strides must be >= dim and multiples of 8");
    if (dtype != DART_FP32 && dtype != DART_BF16)
        return fail(DART_ERR_INVALID_ARG, "dtype must be DART_FP32 or DART_BF16 (got %d)", dtype);
    if (!(eps > 0.0f)) return fail(DART_ERR_INVALID_ARG, "eps must be > 0");
    REQUIRE_PTR(y);
    REQUIRE_PTR(z);
    REQUIRE_PTR(dout);
    REQUIRE_PTR(dy);
    REQUIRE_PTR(dz);
    REQUIRE_PTR(workspace);
    if (((uintptr_t)y | (uintptr_t)z | (uintptr_t)dout | (uintptr_t)dy | (uintptr_t)dz) % 32 != 0)
        return fail(DART_ERR_INVALID_ARG, "y, z, dout, dy and dz must be 32-byte aligned");
    const size_t need = dart::gated_rmsnorm_bwd_workspace_bytes(rows, dim);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    if ((rows / 16 + 1) * (dim / group) / 4 + 1 > 2147483647LL) return fail(DART_ERR_UNSUPPORTED, "too many rows");
    return hip_status(dart::launch_gated_rmsnorm_bwd(dtype, rows, dim, group, y, z, z_row_stride,
                                                     weight, eps, dout, dy, dz, dz_row_stride,
                                                     dweight, workspace, (hipStream_t)stream),
                      "dart_gated_rmsnorm_bwd launch");
}

size_t dart_decode_workspace_bytes(const dart_dims* dims) {
    dart::Shape s;
    if (make_shape(dims, false, s) != DART_OK) return 0;
    if (s.Mcap < 1) return 0;
    return dart::decode_workspace_bytes(s);
}

dart_status dart_decode_step(const dart_dims* dims, const dart_sma_opts* opts, int64_t pos,
                             const void* x, const float* dt, const float* A, const void* Bm,
                             const void* Cm, const void* q, const void* e, const void* z,
                             float* h_state, float* chunk_acc, void* mem_cache, void* y,
                             void* workspace, size_t workspace_bytes, void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, false, s);
    if (st != DART_OK) return st;
    st = check_opts(opts);
    if (st != DART_OK) return st;
    if (s.Mcap < 1) return fail(DART_ERR_INVALID_ARG, "decode needs mem_capacity >= 1");
    if (pos < 0) return fail(DART_ERR_INVALID_ARG, "pos must be >= 0 (got %lld)", (long long)pos);
    const int64_t m = pos / s.S;
    if (m > s.Mcap)
        return fail(DART_ERR_INVALID_ARG, "pos %lld needs %lld cached memories > capacity %lld",
                    (long long)pos, (long long)m, (long long)s.Mcap);
    if (pos % s.S == s.S - 1 && m >= s.Mcap)
        return fail(DART_ERR_INVALID_ARG, "pos %lld closes chunk %lld but the cache holds %lld memories",
                    (long long)pos, (long long)m, (long long)s.Mcap);
    REQUIRE_PTR(x);
    REQUIRE_PTR(dt);
    REQUIRE_PTR(A);
    REQUIRE_PTR(Bm);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(q);
    REQUIRE_PTR(e);
    REQUIRE_PTR(z);
    REQUIRE_PTR(h_state);
    REQUIRE_PTR(chunk_acc);
    REQUIRE_PTR(mem_cache);
    REQUIRE_PTR(y);
    REQUIRE_PTR(workspace);
    const size_t need = dart::decode_workspace_bytes(s);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    const dart::SmaArgs a = sma_args(opts);
    return hip_status(dart::launch_decode(s, a, pos, nullptr, x, dt, A, Bm, Cm, q, e, z, h_state,
                                          chunk_acc, mem_cache, y, workspace, (hipStream_t)stream),
                      "dart_decode_step launch");
}

dart_status dart_decode_step_noalloc(const dart_dims* dims, const dart_sma_opts* opts, int64_t pos,
                                     const void* x, const float* dt, const float* A,
                                     const void* Bm, const void* Cm, const void* q, const void* e,
                                     const void* z, float* h_state, float* chunk_acc,
                                     void* mem_cache, void* y, void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, false, s);
    if (st != DART_OK) return st;
    st = check_opts(opts);
    if (st != DART_OK) return st;
    if (s.Mcap < 1) return fail(DART_ERR_INVALID_ARG, "decode needs mem_capacity >= 1");
    if (pos < 0) return fail(DART_ERR_INVALID_ARG, "pos must be >= 0 (got %lld)", (long long)pos);
    const int64_t m = pos / s.S;
    if (m > s.Mcap)
        return fail(DART_ERR_INVALID_ARG, "pos %lld needs %lld cached memories > capacity %lld",
                    (long long)pos, (long long)m, (long long)s.Mcap);
    if (pos % s.S == s.S - 1 && m >= s.Mcap)
        return fail(DART_ERR_INVALID_ARG, "pos %lld closes chunk %lld but the cache holds %lld memories",
                    (long long)pos, (long long)m, (long long)s.Mcap);
    REQUIRE_PTR(x);
    REQUIRE_PTR(dt);
    REQUIRE_PTR(A);
    REQUIRE_PTR(Bm);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(q);
    REQUIRE_PTR(e);
    REQUIRE_PTR(z);
    REQUIRE_PTR(h_state);
    REQUIRE_PTR(chunk_acc);
    REQUIRE_PTR(mem_cache);
    REQUIRE_PTR(y);
    const size_t need = dart::decode_noalloc_scratch_bytes(s, pos);
    if (need > (size_t)DART_DECODE_NOALLOC_SCRATCH_BYTES)
        return fail(DART_ERR_UNSUPPORTED,
                    "this step needs %zu bytes of scratch; the library's fixed scratch holds %zu "
                    "(use dart_decode_step with a workspace)",
                    need, (size_t)DART_DECODE_NOALLOC_SCRATCH_BYTES);
    const dart::SmaArgs a = sma_args(opts);
    return hip_status(dart::launch_decode_noalloc(s, a, pos, x, dt, A, Bm, Cm, q, e, z, h_state,
                                                  chunk_acc, mem_cache, y, (hipStream_t)stream),
                      "dart_decode_step_noalloc launch");
}

dart_status dart_decode_step_ragged(const dart_dims* dims, const dart_sma_opts* opts,
                                    const int64_t* pos, int64_t pos_max, const void* x,
                                    const float* dt, const float* A, const void* Bm,
                                    const void* Cm, const void* q, const void* e, const void* z,
                                    float* h_state, float* chunk_acc, void* mem_cache, void* y,
                                    void* workspace, size_t workspace_bytes, void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, false, s);
    if (st != DART_OK) return st;
    st = check_opts(opts);
    if (st != DART_OK) return st;
    if (s.Mcap < 1) return fail(DART_ERR_INVALID_ARG, "decode needs mem_capacity >= 1");
    if (pos_max < 0)
        return fail(DART_ERR_INVALID_ARG, "pos_max must be >= 0 (got %lld)", (long long)pos_max);
    if (pos_max >= s.Mcap * s.S)
        return fail(DART_ERR_INVALID_ARG,
                    "pos_max %lld needs more than the %lld memories the cache holds",
                    (long long)pos_max, (long long)s.Mcap);
    REQUIRE_PTR(pos);
    REQUIRE_PTR(x);
    REQUIRE_PTR(dt);
    REQUIRE_PTR(A);
    REQUIRE_PTR(Bm);
    REQUIRE_PTR(Cm);
    REQUIRE_PTR(q);
    REQUIRE_PTR(e);
    REQUIRE_PTR(z);
    REQUIRE_PTR(h_state);
    REQUIRE_PTR(chunk_acc);
    REQUIRE_PTR(mem_cache);
    REQUIRE_PTR(y);
    REQUIRE_PTR(workspace);
    const size_t need = dart::decode_workspace_bytes(s);
    if (workspace_bytes < need)
        return fail(DART_ERR_INVALID_ARG, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    const dart::SmaArgs a = sma_args(opts);
    return hip_status(dart::launch_decode(s, a, pos_max, pos, x, dt, A, Bm, Cm, q, e, z, h_state,
                                          chunk_acc, mem_cache, y, workspace, (hipStream_t)stream),
                      "dart_decode_step_ragged launch");
}

dart_status dart_decode_handoff(const dart_dims* dims, const int64_t* lengths, const void* mem,
                                const float* h_last, float* h_state, float* chunk_acc,
                                void* stream) {
    dart::Shape s;
    dart_status st = make_shape(dims, false, s);
    if (st != DART_OK) return st;
    if (s.Mcap < 1) return fail(DART_ERR_INVALID_ARG, "handoff needs mem_capacity >= 1");
    REQUIRE_PTR(lengths);
    REQUIRE_PTR(mem);
    REQUIRE_PTR(h_last);
    REQUIRE_PTR(h_state);
    REQUIRE_PTR(chunk_acc);
    return hip_status(dart::launch_decode_handoff(s, mem, h_last, lengths, h_state, chunk_acc,
                                                  (hipStream_t)stream),
                      "dart_decode_handoff launch");
}

int64_t dart_decode_cache_elems(const dart_dims* dims, int64_t context) {
    if (!dims || context < 0 || dims->batch < 1 || dims->nheads < 1 || dims->headdim < 1 ||
        dims->dstate < 1 || dims->chunk < 1)
        return 0;
    const int64_t mems = (context + dims->chunk - 1) / dims->chunk;
    return dims->batch * mems * dims->nheads * (int64_t)dims->dstate * dims->headdim;
}

const char* dart_status_string(dart_status status) {
    switch (status) {
        case DART_OK: return "DART_OK";
        case DART_ERR_INVALID_ARG: return "DART_ERR_INVALID_ARG";
        case DART_ERR_UNSUPPORTED: return "DART_ERR_UNSUPPORTED";
        case DART_ERR_HIP: return "DART_ERR_HIP";
    }
    return "DART_ERR_UNKNOWN";
}

const char* dart_last_error(void) { return g_err; }

}  // extern "C"
