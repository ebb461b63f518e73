// C-ABI layer of libblockcopy: argument validation, status codes, thread-local
// error text, the persistent-buffer registry and kernel dispatch. Every check runs
// before anything is enqueued; kernels are launched on the caller's stream.
#include <math.h>
#include <algorithm>
#include <cmath>
#include <vector>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <set>
#include <string>

#include "../../include/bc.h"
#include "bc_internal.h"

using bc::LayerGeom;

namespace {

thread_local std::string g_err;

bc_status fail(bc_status s, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

bc_status ok()
{
    g_err.clear();
    return BC_OK;
}

bc_status hip_fail(hipError_t e, const char *what)
{
    return fail(BC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int esize_of(int32_t dtype) { return dtype == BC_F32 ? 4 : 2; }

bool valid_dtype(int32_t d) { return d == BC_F32 || d == BC_BF16 || d == BC_F16; }
bool valid_layout(int32_t l) { return l == BC_NCHW || l == BC_NHWC; }

size_t tensor_bytes(const bc_tensor &t)
{
    return (size_t)t.n * t.c * t.h * t.w * esize_of(t.dtype);
}

bc_status check_tensor(const bc_tensor &t, const char *name)
{
    if (t.n <= 0 || t.c <= 0 || t.h <= 0 || t.w <= 0)
        return fail(BC_ERR_SHAPE, "%s: all sizes must be positive (n=%d c=%d h=%d w=%d)", name,
                    t.n, t.c, t.h, t.w);
    if (!valid_dtype(t.dtype)) return fail(BC_ERR_DTYPE, "%s: unknown dtype %d", name, t.dtype);
    if (!valid_layout(t.layout)) return fail(BC_ERR_LAYOUT, "%s: unknown layout %d", name, t.layout);
    if ((double)t.n * t.c * t.h * t.w > 4.0e9)
        return fail(BC_ERR_SHAPE, "%s: more than 4e9 elements", name);
    return BC_OK;
}

bool overlap(const void *a, size_t na, const void *b, size_t nb)
{
    if (!a || !b || !na || !nb) return false;
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

// index arguments: both NULL = every block; otherwise both required + capacity
bc_status check_index(const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                      int total_blocks)
{
    if ((d_idx == nullptr) != (d_count == nullptr))
        return fail(BC_ERR_NULL, "d_idx and d_count must both be given or both be NULL");
    if (d_idx && capacity < total_blocks)
        return fail(BC_ERR_CAPACITY, "capacity %d < n*grid_h*grid_w = %d", capacity, total_blocks);
    return BC_OK;
}

// Output blocks of `out` on grid g.
bc_status block_geom(const bc_tensor &out, bc_grid g, LayerGeom &L)
{
    if (g.grid_h <= 0 || g.grid_w <= 0)
        return fail(BC_ERR_SHAPE, "grid must be positive (%d x %d)", g.grid_h, g.grid_w);
    if (out.h % g.grid_h || out.w % g.grid_w)
        return fail(BC_ERR_NOT_DIVISIBLE, "output %d x %d not divisible by the %d x %d block grid",
                    out.h, out.w, g.grid_h, g.grid_w);
    if ((double)out.n * g.grid_h * g.grid_w > (double)(1 << 20))
        return fail(BC_ERR_SHAPE, "more than 2^20 blocks");
    L.gh = g.grid_h;
    L.gw = g.grid_w;
    L.bh = out.h / g.grid_h;
    L.bw = out.w / g.grid_w;
    L.total_blocks = out.n * g.grid_h * g.grid_w;
    return BC_OK;
}

bc_status check_geom(const bc_conv *c, bool conv)
{
    if (c->kh < 1 || c->kw < 1 || c->stride < 1 || c->pad < 0)
        return fail(BC_ERR_SHAPE, "kernel %dx%d, stride %d, pad %d: kernel and stride must be "
                                  ">= 1, pad >= 0", c->kh, c->kw, c->stride, c->pad);
    if (conv && c->relu != 0 && c->relu != 1) return fail(BC_ERR_SHAPE, "relu must be 0 or 1");
    return BC_OK;
}

int conv_out(int in, int k, int s, int p) { return in + 2 * p - k < 0 ? 0 : (in + 2 * p - k) / s + 1; }

// ---------------------------------------------------------------- buffer registry

std::mutex g_mu;
std::set<bc_buffer> g_buffers;
std::map<uintptr_t, bc_buffer> g_by_addr;

}  // namespace

struct bc_buffer_s {
    void *mem;
    bc_tensor desc;
    size_t bytes;
    int valid;
};

namespace {

// Registered buffer that starts at d_out (nullptr if none).
bc_buffer lookup_locked(const void *d_out)
{
    auto it = g_by_addr.find((uintptr_t)d_out);
    return it == g_by_addr.end() ? nullptr : it->second;
}

bc_status check_registered(const void *d_out, const bc_tensor &out, bool sparse)
{
    std::lock_guard<std::mutex> lk(g_mu);
    bc_buffer b = lookup_locked(d_out);
    if (!b) return BC_OK;
    if (memcmp(&b->desc, &out, sizeof out) != 0)
        return fail(BC_ERR_SHAPE, "output descriptor differs from the registered buffer's");
    if (sparse && !b->valid)
        return fail(BC_ERR_UNINITIALIZED,
                    "sparse write into a registered buffer that holds no complete frame yet "
                    "(run a full frame first)");
    return BC_OK;
}

void mark_full(const void *d_out)
{
    std::lock_guard<std::mutex> lk(g_mu);
    bc_buffer b = lookup_locked(d_out);
    if (b) b->valid = 1;
}

}  // namespace

extern "C" {

int32_t bc_abi_version(void) { return BC_ABI_VERSION; }

const char *bc_status_str(int32_t s)
{
    switch (s) {
    case BC_OK: return "ok";
    case BC_ERR_NULL: return "null pointer";
    case BC_ERR_SHAPE: return "inconsistent shape";
    case BC_ERR_DTYPE: return "dtype mismatch";
    case BC_ERR_LAYOUT: return "layout mismatch";
    case BC_ERR_NOT_DIVISIBLE: return "size not divisible by the block grid";
    case BC_ERR_CAPACITY: return "capacity too small";
    case BC_ERR_ALIAS: return "output overlaps an input";
    case BC_ERR_UNINITIALIZED: return "sparse write into an invalid buffer";
    case BC_ERR_UNSUPPORTED: return "unsupported configuration";
    case BC_ERR_HIP: return "HIP runtime error";
    case BC_ERR_CAPTURE: return "allocation refused while the stream is capturing";
    default: return "unknown status";
    }
}

const char *bc_last_error(void) { return g_err.c_str(); }

bc_status bc_build_block_index(const uint8_t *d_mask, int32_t n, bc_grid g, int32_t *d_idx,
                               int32_t capacity, int32_t *d_count, int32_t *h_count,
                               void *stream)
{
    if (!d_mask || !d_idx || !d_count) return fail(BC_ERR_NULL, "d_mask, d_idx and d_count are required");
    if (n <= 0 || g.grid_h <= 0 || g.grid_w <= 0)
        return fail(BC_ERR_SHAPE, "n and grid must be positive");
    const double total = (double)n * g.grid_h * g.grid_w;
    if (total > (double)(1 << 20)) return fail(BC_ERR_SHAPE, "more than 2^20 blocks");
    if (capacity < (int)total)
        return fail(BC_ERR_CAPACITY, "capacity %d < n*grid_h*grid_w = %d", capacity, (int)total);
    if (overlap(d_idx, (size_t)capacity * 4, d_count, 4) ||
        overlap(d_mask, (size_t)total, d_idx, (size_t)capacity * 4) ||
        overlap(d_mask, (size_t)total, d_count, 4))
        return fail(BC_ERR_ALIAS, "mask, index and count must not overlap");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = bc::launch_block_index(d_mask, (int)total, d_idx, d_count, s);
    if (e != hipSuccess) return hip_fail(e, "block index launch");
    if (h_count) {
        e = hipMemcpyAsync(h_count, d_count, sizeof(int32_t), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(e, "count copy");
    }
    return ok();
}

static bc_status gs_common(const bc_tensor &t, bc_grid g, const bc_conv *geom, bool gather,
                           const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                           LayerGeom &L)
{
    bc_status st = check_tensor(t, gather ? "src" : "dst");
    if (st) return st;
    if (gather) {
        if (!geom) return fail(BC_ERR_NULL, "geom is required");
        if ((st = check_geom(geom, false))) return st;
        if (geom->stride > 2 || geom->kh > 7 || geom->kw > 7)
            return fail(BC_ERR_UNSUPPORTED, "gather: stride must be 1 or 2 and kernel edges <= 7");
        bc_tensor out = t;
        out.h = conv_out(t.h, geom->kh, geom->stride, geom->pad);
        out.w = conv_out(t.w, geom->kw, geom->stride, geom->pad);
        if (out.h <= 0 || out.w <= 0) return fail(BC_ERR_SHAPE, "geometry gives an empty output");
        if ((st = block_geom(out, g, L))) return st;
        L.n = t.n; L.cin = t.c; L.hin = t.h; L.win = t.w;
        L.cout = t.c; L.hout = out.h; L.wout = out.w;
        L.kh = geom->kh; L.kw = geom->kw; L.stride = geom->stride; L.pad = geom->pad;
    } else {
        if ((st = block_geom(t, g, L))) return st;
        L.n = t.n; L.cin = L.cout = t.c; L.hin = L.hout = t.h; L.win = L.wout = t.w;
        L.kh = L.kw = L.stride = 1; L.pad = 0;
    }
    if ((st = check_index(d_idx, d_count, capacity, L.total_blocks))) return st;
    L.idx = d_idx;
    L.count = d_count;
    return BC_OK;
}

static int packed_capacity(const int32_t *d_idx, int32_t capacity, int total)
{
    return d_idx ? capacity : total;
}

bc_status bc_gather_halo(const void *d_src, bc_tensor src, bc_grid g, const bc_conv *geom,
                         float pad_value, const int32_t *d_idx, const int32_t *d_count,
                         int32_t capacity, void *d_packed, void *stream)
{
    if (!d_src || !d_packed) return fail(BC_ERR_NULL, "d_src and d_packed are required");
    LayerGeom L;
    bc_status st = gs_common(src, g, geom, true, d_idx, d_count, capacity, L);
    if (st) return st;
    const int es = esize_of(src.dtype);
    const size_t th = (size_t)(L.bh - 1) * L.stride + L.kh, tw = (size_t)(L.bw - 1) * L.stride + L.kw;
    const size_t packed_bytes =
        (size_t)packed_capacity(d_idx, capacity, L.total_blocks) * th * tw * src.c * es;
    if (overlap(d_packed, packed_bytes, d_src, tensor_bytes(src)))
        return fail(BC_ERR_ALIAS, "d_packed overlaps d_src");
    uint32_t bits;
    if (src.dtype == BC_F32) {
        memcpy(&bits, &pad_value, 4);
    } else if (src.dtype == BC_BF16) {
        uint32_t u;
        memcpy(&u, &pad_value, 4);
        if ((u & 0x7FFFFFFFu) > 0x7F800000u) bits = (u >> 16) | 0x40u;
        else bits = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    } else {
        _Float16 h = (_Float16)pad_value;
        uint16_t hb;
        memcpy(&hb, &h, 2);
        bits = hb;
    }
    hipError_t e = bc::launch_gather_halo(d_src, es, src.layout == BC_NHWC, L, bits, d_packed,
                                          (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "gather launch");
    return ok();
}

bc_status bc_scatter_blocks(const void *d_packed, const int32_t *d_idx, const int32_t *d_count,
                            int32_t capacity, bc_grid g, void *d_dst, bc_tensor dst, void *stream)
{
    if (!d_packed || !d_dst) return fail(BC_ERR_NULL, "d_packed and d_dst are required");
    LayerGeom L;
    bc_status st = gs_common(dst, g, nullptr, false, d_idx, d_count, capacity, L);
    if (st) return st;
    const int es = esize_of(dst.dtype);
    const size_t packed_bytes = (size_t)packed_capacity(d_idx, capacity, L.total_blocks) * L.bh *
                                L.bw * dst.c * es;
    if (overlap(d_packed, packed_bytes, d_dst, tensor_bytes(dst)))
        return fail(BC_ERR_ALIAS, "d_dst overlaps d_packed");
    if (d_idx && overlap(d_dst, tensor_bytes(dst), d_idx, (size_t)capacity * 4))
        return fail(BC_ERR_ALIAS, "d_dst overlaps the index");
    hipError_t e = bc::launch_scatter_blocks(d_packed, es, dst.layout == BC_NHWC, L, d_dst,
                                             (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "scatter launch");
    return ok();
}

// Validation shared by the conv and pooling layers.
static bc_status layer_common(const bc_conv *geom, bool conv, const void *d_in, const bc_tensor &in,
                              void *d_out, const bc_tensor &out, bc_grid g, const int32_t *d_idx,
                              const int32_t *d_count, int32_t capacity, LayerGeom &L)
{
    if (!geom || !d_in || !d_out) return fail(BC_ERR_NULL, "geometry, d_in and d_out are required");
    bc_status st;
    if ((st = check_geom(geom, conv))) return st;
    if ((st = check_tensor(in, "in"))) return st;
    if ((st = check_tensor(out, "out"))) return st;
    if (in.dtype != out.dtype) return fail(BC_ERR_DTYPE, "in and out dtypes differ");
    if (in.layout != out.layout) return fail(BC_ERR_LAYOUT, "in and out layouts differ");
    if (in.layout == BC_NHWC && in.dtype == BC_F32)
        return fail(BC_ERR_UNSUPPORTED, "channels-last layers take BF16 or F16");
    if (in.layout == BC_NCHW && in.dtype != BC_F32)
        return fail(BC_ERR_UNSUPPORTED, "channels-first layers take F32");
    if (out.n != in.n) return fail(BC_ERR_SHAPE, "out.n %d != in.n %d", out.n, in.n);
    const int oh = conv_out(in.h, geom->kh, geom->stride, geom->pad);
    const int ow = conv_out(in.w, geom->kw, geom->stride, geom->pad);
    if (out.h != oh || out.w != ow)
        return fail(BC_ERR_SHAPE, "out is %dx%d but the geometry gives %dx%d", out.h, out.w, oh, ow);
    if ((st = block_geom(out, g, L))) return st;
    if ((st = check_index(d_idx, d_count, capacity, L.total_blocks))) return st;
    if (overlap(d_out, tensor_bytes(out), d_in, tensor_bytes(in)))
        return fail(BC_ERR_ALIAS, "d_out overlaps d_in");
    if (d_idx && (overlap(d_out, tensor_bytes(out), d_idx, (size_t)capacity * 4) ||
                  overlap(d_out, tensor_bytes(out), d_count, 4)))
        return fail(BC_ERR_ALIAS, "d_out overlaps the index");
    L.n = in.n; L.cin = in.c; L.hin = in.h; L.win = in.w;
    L.cout = out.c; L.hout = out.h; L.wout = out.w;
    L.kh = geom->kh; L.kw = geom->kw; L.stride = geom->stride; L.pad = geom->pad;
    L.idx = d_idx;
    L.count = d_count;
    return BC_OK;
}

namespace {

// Every check of one convolution call, before anything is enqueued.
bc_status conv_checks(const bc_conv *conv, const void *d_in, const bc_tensor &in, const void *d_w,
                      const float *d_bias, const void *d_residual, void *d_out,
                      const bc_tensor &out, const bc_grid &g, const int32_t *d_idx,
                      const int32_t *d_count, int32_t capacity, LayerGeom &L)
{
    if (!d_w) return fail(BC_ERR_NULL, "d_w is required");
    bc_status st = layer_common(conv, true, d_in, in, d_out, out, g, d_idx, d_count, capacity, L);
    if (st) return st;
    const size_t wbytes = (size_t)out.c * in.c * conv->kh * conv->kw * esize_of(in.dtype);
    const size_t obytes = tensor_bytes(out);
    if (overlap(d_out, obytes, d_w, wbytes)) return fail(BC_ERR_ALIAS, "d_out overlaps d_w");
    if (overlap(d_out, obytes, d_residual, obytes)) return fail(BC_ERR_ALIAS, "d_out overlaps d_residual");
    if (overlap(d_out, obytes, d_bias, (size_t)out.c * 4)) return fail(BC_ERR_ALIAS, "d_out overlaps d_bias");
    const char *why = "";
    if (in.layout == BC_NHWC) {
        if (!bc::conv_nhwc_mfma_supported(L, &why)) return fail(BC_ERR_UNSUPPORTED, "%s", why);
    } else {
        const int th = (L.bh - 1) * L.stride + L.kh, tw = (L.bw - 1) * L.stride + L.kw;
        if (L.bh * L.bw > 2048 || (th * tw + L.kh * L.kw) * 4 > 48 * 1024)
            return fail(BC_ERR_UNSUPPORTED, "fp32 path: output blocks above 2048 pixels or halo "
                                            "tiles above 48 KB per channel");
    }
    return check_registered(d_out, out, d_idx != nullptr);
}

// Status of a failed convolution launch: a refused capture, a shape the kernels do not
// take (with the reason), or a HIP error.
bc_status conv_fail(hipError_t e, const char *why, const char *what)
{
    if (e == hipErrorStreamCaptureUnsupported && why && *why) return fail(BC_ERR_CAPTURE, "%s", why);
    if (e == hipErrorInvalidValue && why && *why) return fail(BC_ERR_UNSUPPORTED, "%s", why);
    return hip_fail(e, what);
}

bc_status conv_launch(const bc_conv *conv, const void *d_in, const bc_tensor &in, const void *d_w,
                      const float *d_bias, const void *d_residual, void *d_out,
                      const LayerGeom &L, hipStream_t s, bool noalloc = false)
{
    const char *why = "";
    hipError_t e;
    if (in.layout == BC_NHWC) {
        e = (noalloc ? bc::launch_conv_nhwc_mfma_noalloc : bc::launch_conv_nhwc_mfma)((const uint16_t *)d_in, (const uint16_t *)d_w, d_bias,
                                      (const uint16_t *)d_residual, (uint16_t *)d_out, conv->relu,
                                      in.dtype == BC_BF16 ? bc::Half16::BF16 : bc::Half16::F16, L,
                                      s, &why);
    } else {
        e = bc::launch_conv_nchw_f32((const float *)d_in, (const float *)d_w, d_bias,
                                     (const float *)d_residual, (float *)d_out, conv->relu, L, s,
                                     &why);
    }
    if (e != hipSuccess) return conv_fail(e, why, "conv launch");
    return BC_OK;
}

// Bytes of every tensor one call reads, for the cross-call alias checks.
bool call_reads_overlap(const bc_conv_call &c, const void *p, size_t bytes)
{
    const size_t wbytes = (size_t)c.out.c * c.in.c * c.conv.kh * c.conv.kw * esize_of(c.in.dtype);
    return overlap(p, bytes, c.d_in, tensor_bytes(c.in)) || overlap(p, bytes, c.d_w, wbytes) ||
           overlap(p, bytes, c.d_bias, (size_t)c.out.c * 4) ||
           overlap(p, bytes, c.d_residual, tensor_bytes(c.out)) ||
           overlap(p, bytes, c.d_out, tensor_bytes(c.out));
}

}  // namespace

bc_status bc_sparse_conv2d(const bc_conv *conv, const void *d_in, bc_tensor in, const void *d_w,
                           const float *d_bias, const void *d_residual, void *d_out, bc_tensor out,
                           bc_grid g, const int32_t *d_idx, const int32_t *d_count,
                           int32_t capacity, void *stream)
{
    LayerGeom L;
    bc_status st = conv_checks(conv, d_in, in, d_w, d_bias, d_residual, d_out, out, g, d_idx,
                               d_count, capacity, L);
    if (st) return st;
    if ((st = conv_launch(conv, d_in, in, d_w, d_bias, d_residual, d_out, L, (hipStream_t)stream)))
        return st;
    if (!d_idx) mark_full(d_out);
    return ok();
}

bc_status bc_sparse_conv2d_noalloc(const bc_conv *conv, const void *d_in, bc_tensor in,
                                   const void *d_w, const float *d_bias, const void *d_residual,
                                   void *d_out, bc_tensor out, bc_grid g, const int32_t *d_idx,
                                   const int32_t *d_count, int32_t capacity, void *stream)
{
    LayerGeom L;
    bc_status st = conv_checks(conv, d_in, in, d_w, d_bias, d_residual, d_out, out, g, d_idx,
                               d_count, capacity, L);
    if (st) return st;
    if (in.layout == BC_NHWC) {
        const size_t need = bc::conv_nhwc_split_bytes(L), have = bc::conv_nhwc_scratch_bytes();
        if (need > have)
            return fail(BC_ERR_CAPACITY, "this layer's split-K partials need %zu bytes; the fixed "
                                         "scratch array holds %zu (use bc_sparse_conv2d)", need, have);
    }
    if ((st = conv_launch(conv, d_in, in, d_w, d_bias, d_residual, d_out, L, (hipStream_t)stream,
                          true)))
        return st;
    if (!d_idx) mark_full(d_out);
    return ok();
}

bc_status bc_sparse_conv2d_pair(const bc_conv_call *a, const bc_conv_call *b, bc_grid g,
                                const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                void *stream)
{
    if (!a || !b) return fail(BC_ERR_NULL, "both calls are required");
    LayerGeom La, Lb;
    bc_status st = conv_checks(&a->conv, a->d_in, a->in, a->d_w, a->d_bias, a->d_residual,
                               a->d_out, a->out, g, d_idx, d_count, capacity, La);
    if (st) return st;
    if ((st = conv_checks(&b->conv, b->d_in, b->in, b->d_w, b->d_bias, b->d_residual, b->d_out,
                          b->out, g, d_idx, d_count, capacity, Lb)))
        return st;
    if (call_reads_overlap(*b, a->d_out, tensor_bytes(a->out)))
        return fail(BC_ERR_ALIAS, "the first call's output overlaps a tensor of the second");
    if (call_reads_overlap(*a, b->d_out, tensor_bytes(b->out)))
        return fail(BC_ERR_ALIAS, "the second call's output overlaps a tensor of the first");
    hipStream_t s = (hipStream_t)stream;
    if (a->in.layout == BC_NHWC && b->in.layout == BC_NHWC && a->in.dtype == b->in.dtype) {
        const bc::ConvCall ca{(const uint16_t *)a->d_in, (const uint16_t *)a->d_w,
                              (const uint16_t *)a->d_residual, a->d_bias, (uint16_t *)a->d_out,
                              a->conv.relu, La};
        const bc::ConvCall cb{(const uint16_t *)b->d_in, (const uint16_t *)b->d_w,
                              (const uint16_t *)b->d_residual, b->d_bias, (uint16_t *)b->d_out,
                              b->conv.relu, Lb};
        const char *why = "";
        const hipError_t e = bc::launch_conv_pair_nhwc_mfma(
            ca, cb, a->in.dtype == BC_BF16 ? bc::Half16::BF16 : bc::Half16::F16, s, &why);
        if (e != hipSuccess) return conv_fail(e, why, "conv pair launch");
    } else {
        if ((st = conv_launch(&a->conv, a->d_in, a->in, a->d_w, a->d_bias, a->d_residual, a->d_out,
                              La, s)))
            return st;
        if ((st = conv_launch(&b->conv, b->d_in, b->in, b->d_w, b->d_bias, b->d_residual, b->d_out,
                              Lb, s)))
            return st;
    }
    if (!d_idx) {
        mark_full(a->d_out);
        mark_full(b->d_out);
    }
    return ok();
}

bc_status bc_sparse_spp(const void *d_in, bc_tensor in, const bc_spp_geom *spp, const void *d_w,
                        const float *d_bias, void *d_levels, void *d_out, bc_tensor out, bc_grid g,
                        const int32_t *d_idx, const int32_t *d_count, int32_t capacity, void *stream)
{
    if (!d_in || !spp || !d_w || !d_levels || !d_out)
        return fail(BC_ERR_NULL, "d_in, spp, d_w, d_levels and d_out are required");
    bc_status st;
    if ((st = check_tensor(in, "in"))) return st;
    if ((st = check_tensor(out, "out"))) return st;
    if (in.dtype != out.dtype) return fail(BC_ERR_DTYPE, "in and out dtypes differ");
    if (in.layout != out.layout) return fail(BC_ERR_LAYOUT, "in and out layouts differ");
    if (in.layout != BC_NHWC || in.dtype == BC_F32)
        return fail(BC_ERR_UNSUPPORTED, "pyramid pooling takes channels-last BF16 or F16");
    if (in.c % 8 || in.c > bc::kMaxSppChannels || 256 % (in.c / 8))
        return fail(BC_ERR_UNSUPPORTED, "pyramid pooling needs c %% 8 == 0 with c / 8 dividing 256 "
                                        "(c = %d)", in.c);
    if (spp->levels < 1 || spp->levels > bc::kMaxSppLevels)
        return fail(BC_ERR_SHAPE, "levels must be 1..%d (got %d)", bc::kMaxSppLevels, spp->levels);
    if (spp->cl < 8 || spp->cl > 256 || spp->cl % 8)
        return fail(BC_ERR_SHAPE, "cl must be a multiple of 8 in 8..256 (got %d)", spp->cl);
    bc::SppGeom G;
    G.first[0] = 0;
    for (int l = 0; l < spp->levels; ++l) {
        if (spp->rows[l] < 1 || spp->rows[l] > in.h || spp->cols[l] < 1 || spp->cols[l] > in.w)
            return fail(BC_ERR_SHAPE, "level %d: %d x %d bins on a %d x %d map", l, spp->rows[l],
                        spp->cols[l], in.h, in.w);
        G.rows[l] = spp->rows[l];
        G.cols[l] = spp->cols[l];
        G.first[l + 1] = G.first[l] + spp->rows[l] * spp->cols[l];
    }
    if (out.n != in.n || out.h != in.h || out.w != in.w || out.c != in.c + spp->levels * spp->cl)
        return fail(BC_ERR_SHAPE, "out must be [n][h][w][c + levels * cl] = [%d][%d][%d][%d]", in.n,
                    in.h, in.w, in.c + spp->levels * spp->cl);
    LayerGeom L;
    if ((st = block_geom(out, g, L))) return st;
    if ((st = check_index(d_idx, d_count, capacity, L.total_blocks))) return st;
    const int es = esize_of(in.dtype);
    const size_t wbytes = (size_t)spp->levels * spp->cl * in.c * es;
    const size_t lbytes = (size_t)in.n * G.first[spp->levels] * spp->cl * es;
    const size_t obytes = tensor_bytes(out), ibytes = tensor_bytes(in);
    if (obytes >= ((size_t)1 << 31) || ibytes >= ((size_t)1 << 31) || lbytes >= ((size_t)1 << 31))
        return fail(BC_ERR_UNSUPPORTED, "tensors of 2 GiB or more");
    if (overlap(d_out, obytes, d_in, ibytes)) return fail(BC_ERR_ALIAS, "d_out overlaps d_in");
    if (overlap(d_out, obytes, d_levels, lbytes) || overlap(d_levels, lbytes, d_in, ibytes) ||
        overlap(d_levels, lbytes, d_w, wbytes) || overlap(d_levels, lbytes, d_bias, (size_t)spp->levels * spp->cl * 4))
        return fail(BC_ERR_ALIAS, "d_levels overlaps another tensor");
    if (overlap(d_out, obytes, d_w, wbytes) || overlap(d_out, obytes, d_bias, (size_t)spp->levels * spp->cl * 4))
        return fail(BC_ERR_ALIAS, "d_out overlaps the weights or biases");
    if (d_idx && (overlap(d_out, obytes, d_idx, (size_t)capacity * 4) || overlap(d_out, obytes, d_count, 4) ||
                  overlap(d_levels, lbytes, d_idx, (size_t)capacity * 4) || overlap(d_levels, lbytes, d_count, 4)))
        return fail(BC_ERR_ALIAS, "an output overlaps the index");
    if ((st = check_registered(d_out, out, d_idx != nullptr))) return st;
    G.n = in.n; G.h = in.h; G.w = in.w; G.c = in.c; G.vpp = in.c / 8;
    G.levels = spp->levels; G.cl = spp->cl; G.cout = out.c;
    G.gh = L.gh; G.gw = L.gw; G.bh = L.bh; G.bw = L.bw; G.total_blocks = L.total_blocks;
    G.in_bytes = (int)ibytes; G.w_bytes = (int)wbytes; G.lv_bytes = (int)lbytes; G.out_bytes = (int)obytes;
    hipError_t e = bc::launch_spp((const uint16_t *)d_in, (const uint16_t *)d_w, d_bias,
                                  (uint16_t *)d_levels, (uint16_t *)d_out, G, in.dtype == BC_BF16,
                                  d_idx, d_count, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "pyramid pooling launch");
    if (!d_idx) mark_full(d_out);
    return ok();
}

bc_status bc_sparse_maxpool2d(const bc_conv *geom, const void *d_in, bc_tensor in, void *d_out,
                              bc_tensor out, bc_grid g, const int32_t *d_idx,
                              const int32_t *d_count, int32_t capacity, void *stream)
{
    LayerGeom L;
    bc_status st = layer_common(geom, false, d_in, in, d_out, out, g, d_idx, d_count, capacity, L);
    if (st) return st;
    if (in.c != out.c) return fail(BC_ERR_SHAPE, "pooling keeps the channel count");
    if (in.layout == BC_NHWC && in.c % 8)
        return fail(BC_ERR_UNSUPPORTED, "channels-last pooling needs C % 8 == 0");
    if ((st = check_registered(d_out, out, d_idx != nullptr))) return st;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (in.layout == BC_NHWC)
        e = bc::launch_maxpool_nhwc16((const uint16_t *)d_in, (uint16_t *)d_out,
                                      in.dtype == BC_BF16 ? bc::Half16::BF16 : bc::Half16::F16, L, s);
    else
        e = bc::launch_maxpool_nchw32((const float *)d_in, (float *)d_out, L, s);
    if (e != hipSuccess) return hip_fail(e, "maxpool launch");
    if (!d_idx) mark_full(d_out);
    return ok();
}

bc_status bc_fold_bn(const float *w, int32_t cout, int32_t per_out, const float *conv_bias,
                     const float *gamma, const float *beta, const float *mean, const float *var,
                     float eps, float *w_out, float *b_out)
{
    if (!w || !gamma || !beta || !mean || !var || !w_out || !b_out)
        return fail(BC_ERR_NULL, "w, gamma, beta, mean, var, w_out and b_out are required");
    if (cout <= 0 || per_out <= 0) return fail(BC_ERR_SHAPE, "cout and per_out must be positive");
    for (int co = 0; co < cout; ++co) {
        const double scale = (double)gamma[co] / sqrt((double)var[co] + (double)eps);
        const double cb = conv_bias ? (double)conv_bias[co] : 0.0;
        b_out[co] = (float)((double)beta[co] + (cb - (double)mean[co]) * scale);
        for (int k = 0; k < per_out; ++k) {
            const size_t i = (size_t)co * per_out + k;
            w_out[i] = (float)((double)w[i] * scale);
        }
    }
    return ok();
}

bc_status bc_repack_weights(const float *w_oihw, int32_t cout, int32_t cin, int32_t kh, int32_t kw,
                            int32_t dtype, void *h_out)
{
    if (!w_oihw || !h_out) return fail(BC_ERR_NULL, "w_oihw and h_out are required");
    if (cout <= 0 || cin <= 0 || kh <= 0 || kw <= 0) return fail(BC_ERR_SHAPE, "sizes must be positive");
    if (!valid_dtype(dtype)) return fail(BC_ERR_DTYPE, "unknown dtype %d", dtype);
    for (int co = 0; co < cout; ++co)
        for (int i = 0; i < kh; ++i)
            for (int j = 0; j < kw; ++j)
                for (int ci = 0; ci < cin; ++ci) {
                    const float v = w_oihw[(((size_t)co * cin + ci) * kh + i) * kw + j];
                    const size_t o = (((size_t)co * kh + i) * kw + j) * cin + ci;
                    if (dtype == BC_F32) {
                        ((float *)h_out)[o] = v;
                    } else if (dtype == BC_BF16) {
                        uint32_t u;
                        memcpy(&u, &v, 4);
                        const uint32_t r = ((u & 0x7FFFFFFFu) > 0x7F800000u)
                                               ? ((u >> 16) | 0x40u)
                                               : ((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
                        ((uint16_t *)h_out)[o] = (uint16_t)r;
                    } else {
                        const _Float16 h = (_Float16)v;
                        memcpy((uint16_t *)h_out + o, &h, 2);
                    }
                }
    return ok();
}

bc_status bc_buffer_register(void *d_mem, bc_tensor desc, bc_buffer *out)
{
    if (!d_mem || !out) return fail(BC_ERR_NULL, "d_mem and out are required");
    bc_status st = check_tensor(desc, "desc");
    if (st) return st;
    const size_t bytes = tensor_bytes(desc);
    std::lock_guard<std::mutex> lk(g_mu);
    for (bc_buffer b : g_buffers)
        if (overlap(b->mem, b->bytes, d_mem, bytes))
            return fail(BC_ERR_ALIAS, "memory overlaps an already registered buffer");
    bc_buffer b = new bc_buffer_s{d_mem, desc, bytes, 0};
    g_buffers.insert(b);
    g_by_addr[(uintptr_t)d_mem] = b;
    *out = b;
    return ok();
}

bc_status bc_buffer_release(bc_buffer b)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!b || !g_buffers.count(b)) return fail(BC_ERR_NULL, "unknown buffer handle");
    g_by_addr.erase((uintptr_t)b->mem);
    g_buffers.erase(b);
    delete b;
    return ok();
}

bc_status bc_buffer_invalidate(bc_buffer b)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!b || !g_buffers.count(b)) return fail(BC_ERR_NULL, "unknown buffer handle");
    b->valid = 0;
    return ok();
}

bc_status bc_buffer_mark_written(bc_buffer b, int32_t full_mask)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!b || !g_buffers.count(b)) return fail(BC_ERR_NULL, "unknown buffer handle");
    if (full_mask) {
        b->valid = 1;
        return ok();
    }
    if (!b->valid)
        return fail(BC_ERR_UNINITIALIZED, "sparse write recorded on a buffer with no full frame");
    return ok();
}

int32_t bc_buffer_is_valid(bc_buffer b)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!b || !g_buffers.count(b)) return -1;
    return b->valid;
}

// ---------------------------------------------------------------- policy-side steps

bc_status bc_sample_execution_grid(const float *d_prob, int32_t n, bc_grid g, uint64_t seed,
                                   uint64_t frame, uint8_t *d_mask, int32_t *d_idx,
                                   int32_t capacity, int32_t *d_count, int32_t *h_count,
                                   void *stream)
{
    if (!d_prob || !d_mask || !d_idx || !d_count)
        return fail(BC_ERR_NULL, "d_prob, d_mask, d_idx and d_count are required");
    if (n <= 0 || g.grid_h <= 0 || g.grid_w <= 0)
        return fail(BC_ERR_SHAPE, "n and grid must be positive");
    const double total = (double)n * g.grid_h * g.grid_w;
    if (total > (double)(1 << 20)) return fail(BC_ERR_SHAPE, "more than 2^20 blocks");
    if (capacity < (int)total)
        return fail(BC_ERR_CAPACITY, "capacity %d < n*grid_h*grid_w = %d", capacity, (int)total);
    const size_t nb = (size_t)total;
    if (overlap(d_idx, (size_t)capacity * 4, d_count, 4) || overlap(d_mask, nb, d_idx, (size_t)capacity * 4) ||
        overlap(d_mask, nb, d_count, 4) || overlap(d_prob, nb * 4, d_mask, nb) ||
        overlap(d_prob, nb * 4, d_idx, (size_t)capacity * 4) || overlap(d_prob, nb * 4, d_count, 4))
        return fail(BC_ERR_ALIAS, "probabilities, mask, index and count must not overlap");
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = bc::launch_sample_index(d_prob, (int)total, seed, frame, d_mask, d_idx, d_count, s);
    if (e != hipSuccess) return hip_fail(e, "sampling launch");
    if (h_count) {
        e = hipMemcpyAsync(h_count, d_count, sizeof(int32_t), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_fail(e, "count copy");
    }
    return ok();
}

bc_status bc_update_frame_state(const void *d_frame, void *d_state, bc_tensor desc, bc_grid g,
                                const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                void *stream)
{
    if (!d_frame || !d_state) return fail(BC_ERR_NULL, "d_frame and d_state are required");
    bc_status st = check_tensor(desc, "desc");
    if (st) return st;
    LayerGeom L;
    if ((st = block_geom(desc, g, L))) return st;
    if ((st = check_index(d_idx, d_count, capacity, L.total_blocks))) return st;
    const size_t bytes = tensor_bytes(desc);
    if (overlap(d_frame, bytes, d_state, bytes)) return fail(BC_ERR_ALIAS, "frame and state overlap");
    if (d_idx && (overlap(d_idx, (size_t)capacity * 4, d_state, bytes) || overlap(d_count, 4, d_state, bytes)))
        return fail(BC_ERR_ALIAS, "the index overlaps the state");
    hipError_t e = bc::launch_frame_state(d_frame, d_state, desc.n, desc.c, desc.h, desc.w,
                                          esize_of(desc.dtype), desc.layout == BC_NHWC, g.grid_h,
                                          g.grid_w, d_idx, d_count, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "frame state launch");
    return ok();
}

bc_status bc_seg_information_gain(const void *d_logits, const void *d_prev_logits,
                                  bc_tensor desc, int32_t classes, bc_grid g,
                                  const uint8_t *d_mask, float *d_ig, void *stream)
{
    if (!d_logits || !d_prev_logits || !d_ig)
        return fail(BC_ERR_NULL, "d_logits, d_prev_logits and d_ig are required");
    bc_status st = check_tensor(desc, "desc");
    if (st) return st;
    if (desc.layout == BC_NCHW && desc.dtype != BC_F32)
        return fail(BC_ERR_DTYPE, "channels-first scores must be float32");
    if (desc.layout == BC_NHWC && desc.dtype == BC_F32)
        return fail(BC_ERR_DTYPE, "channels-last scores must be bf16 or f16");
    if (desc.layout == BC_NHWC && desc.c % 8)
        return fail(BC_ERR_UNSUPPORTED, "channels-last scores need C %% 8 == 0 (got %d)", desc.c);
    if (classes < 1 || classes > desc.c)
        return fail(BC_ERR_SHAPE, "classes %d outside 1..%d (the channel count)", classes, desc.c);
    if (classes > 32) return fail(BC_ERR_UNSUPPORTED, "at most 32 classes (got %d)", classes);
    LayerGeom L;
    if ((st = block_geom(desc, g, L))) return st;
    const int es = esize_of(desc.dtype);
    const double img_bytes = (double)es * desc.c * desc.h * desc.w;
    if (img_bytes >= 2147483392.0) return fail(BC_ERR_UNSUPPORTED, "one image's scores must be < 2 GiB");
    const size_t bytes = tensor_bytes(desc), igb = (size_t)L.total_blocks * 4;
    if (overlap(d_ig, igb, d_logits, bytes) || overlap(d_ig, igb, d_prev_logits, bytes) ||
        overlap(d_ig, igb, d_mask, (size_t)L.total_blocks))
        return fail(BC_ERR_ALIAS, "d_ig overlaps an input");
    hipError_t e = bc::launch_seg_information_gain(
        d_logits, d_prev_logits, desc.n, desc.c, classes, desc.h, desc.w, es,
        desc.layout == BC_NHWC, desc.dtype == BC_BF16, g.grid_h, g.grid_w, d_mask, d_ig,
        (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "information gain launch");
    return ok();
}

bc_status bc_sparse_upsample_add(const void *d_coarse, bc_tensor coarse, const void *d_skip,
                                 void *d_out, bc_tensor out, bc_grid g, int32_t relu,
                                 const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                 void *stream)
{
    if (!d_coarse || !d_out) return fail(BC_ERR_NULL, "d_coarse and d_out are required");
    bc_status st;
    if ((st = check_tensor(coarse, "coarse"))) return st;
    if ((st = check_tensor(out, "out"))) return st;
    if (coarse.dtype != out.dtype) return fail(BC_ERR_DTYPE, "coarse and out dtypes differ");
    if (coarse.layout != out.layout) return fail(BC_ERR_LAYOUT, "coarse and out layouts differ");
    if (out.layout == BC_NHWC && out.dtype == BC_F32)
        return fail(BC_ERR_UNSUPPORTED, "channels-last maps take BF16 or F16");
    if (out.layout == BC_NCHW && out.dtype != BC_F32)
        return fail(BC_ERR_UNSUPPORTED, "channels-first maps take F32");
    if (out.layout == BC_NHWC && out.c % 8)
        return fail(BC_ERR_UNSUPPORTED, "channels-last maps need C %% 8 == 0 (got %d)", out.c);
    if (out.n != coarse.n || out.c != coarse.c || out.h != 2 * coarse.h || out.w != 2 * coarse.w)
        return fail(BC_ERR_SHAPE, "out must be [n][c][2h][2w] of coarse's [n][c][h][w]");
    if (relu != 0 && relu != 1) return fail(BC_ERR_SHAPE, "relu must be 0 or 1");
    LayerGeom L;
    if ((st = block_geom(out, g, L))) return st;
    if ((st = check_index(d_idx, d_count, capacity, L.total_blocks))) return st;
    const size_t ob = tensor_bytes(out), cb = tensor_bytes(coarse);
    if (out.layout == BC_NHWC) {
        if (ob >= 2147483392u) return fail(BC_ERR_UNSUPPORTED, "channels-last out must be < 2 GiB");
        const double chunks = ceil((double)L.bh * L.bw * (out.c / 8) / 256.0);
        if (chunks * L.total_blocks >= 4194304.0)
            return fail(BC_ERR_UNSUPPORTED, "too many workgroups (blocks x block size)");
    }
    if (overlap(d_out, ob, d_coarse, cb)) return fail(BC_ERR_ALIAS, "d_out overlaps d_coarse");
    if (overlap(d_out, ob, d_skip, ob)) return fail(BC_ERR_ALIAS, "d_out overlaps d_skip");
    if (d_idx && (overlap(d_out, ob, d_idx, (size_t)capacity * 4) || overlap(d_out, ob, d_count, 4)))
        return fail(BC_ERR_ALIAS, "d_out overlaps the index");
    if ((st = check_registered(d_out, out, d_idx != nullptr))) return st;
    hipError_t e = bc::launch_upsample_add(d_coarse, d_skip, d_out, out.n, out.c, coarse.h,
                                           coarse.w, esize_of(out.dtype), out.layout == BC_NHWC,
                                           out.dtype == BC_BF16, g.grid_h, g.grid_w, d_idx,
                                           d_count, relu, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "upsample launch");
    if (!d_idx) mark_full(d_out);
    return ok();
}

bc_status bc_policy_input(const void *d_frame, const void *d_state, bc_tensor frame,
                          const void *d_scores, bc_tensor scores, int32_t classes,
                          const uint8_t *d_prev_mask, bc_grid g, void *d_out, bc_tensor out,
                          void *stream)
{
    if (!d_frame || !d_state || !d_scores || !d_out)
        return fail(BC_ERR_NULL, "d_frame, d_state, d_scores and d_out are required");
    bc_status st;
    if ((st = check_tensor(frame, "frame"))) return st;
    if ((st = check_tensor(scores, "scores"))) return st;
    if ((st = check_tensor(out, "out"))) return st;
    if (frame.layout != BC_NHWC || scores.layout != BC_NHWC || out.layout != BC_NHWC)
        return fail(BC_ERR_LAYOUT, "frame, scores and out must be channels last (NHWC)");
    if (frame.dtype == BC_F32 || scores.dtype != frame.dtype || out.dtype != frame.dtype)
        return fail(BC_ERR_DTYPE, "frame, scores and out must share one 16-bit dtype");
    if (frame.c != 3) return fail(BC_ERR_SHAPE, "frame must have 3 channels (got %d)", frame.c);
    if (frame.h % 4 || frame.w % 4) return fail(BC_ERR_SHAPE, "frame size must be a multiple of 4");
    const int h4 = frame.h / 4, w4 = frame.w / 4;
    if (scores.n != frame.n || scores.h != h4 || scores.w != w4)
        return fail(BC_ERR_SHAPE, "scores must be [n][h/4][w/4][c] of the frame");
    if (scores.c % 8) return fail(BC_ERR_UNSUPPORTED, "score channels must be a multiple of 8");
    if (classes < 1 || classes > scores.c || classes > 24)
        return fail(BC_ERR_SHAPE, "classes %d outside 1..min(24, %d)", classes, scores.c);
    if (out.n != frame.n || out.h != h4 || out.w != w4 || out.c != 32)
        return fail(BC_ERR_SHAPE, "out must be [n][h/4][w/4][32]");
    if (g.grid_h <= 0 || g.grid_w <= 0 || h4 % g.grid_h || w4 % g.grid_w)
        return fail(BC_ERR_NOT_DIVISIBLE, "the quarter-resolution map is not divisible by the grid");
    if (tensor_bytes(frame) >= 2147483392u)
        return fail(BC_ERR_UNSUPPORTED, "frame must be below 2 GiB");
    const size_t ob = tensor_bytes(out);
    if (overlap(d_out, ob, d_frame, tensor_bytes(frame)) || overlap(d_out, ob, d_state, tensor_bytes(frame)) ||
        overlap(d_out, ob, d_scores, tensor_bytes(scores)) ||
        overlap(d_out, ob, d_prev_mask, (size_t)frame.n * g.grid_h * g.grid_w))
        return fail(BC_ERR_ALIAS, "d_out overlaps an input");
    hipError_t e = bc::launch_policy_input(d_frame, d_state, d_scores, d_prev_mask, d_out, frame.n,
                                           frame.h, frame.w, scores.c, classes, g.grid_h, g.grid_w,
                                           frame.dtype == BC_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "policy input launch");
    return ok();
}

bc_status bc_policy_probabilities(const void *d_logits, bc_tensor logits, float *d_prob,
                                  void *stream)
{
    if (!d_logits || !d_prob) return fail(BC_ERR_NULL, "d_logits and d_prob are required");
    bc_status st = check_tensor(logits, "logits");
    if (st) return st;
    if (logits.layout != BC_NHWC) return fail(BC_ERR_LAYOUT, "logits must be channels last");
    if (logits.dtype == BC_F32) return fail(BC_ERR_DTYPE, "logits must be bf16 or f16");
    const double blocks = (double)logits.n * logits.h * logits.w;
    if (blocks > (double)(1 << 20)) return fail(BC_ERR_SHAPE, "more than 2^20 blocks");
    if (overlap(d_prob, (size_t)blocks * 4, d_logits, tensor_bytes(logits)))
        return fail(BC_ERR_ALIAS, "d_prob overlaps d_logits");
    hipError_t e = bc::launch_policy_probabilities(d_logits, (int)blocks, logits.c,
                                                   logits.dtype == BC_BF16, d_prob, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "policy probabilities launch");
    return ok();
}

// ---------------------------------------------------------------- policy training

static bc_status check_grad_map(const bc_tensor &t, const char *name)
{
    bc_status st = check_tensor(t, name);
    if (st) return st;
    if (t.layout != BC_NHWC) return fail(BC_ERR_LAYOUT, "%s must be channels last", name);
    if (t.dtype == BC_F32) return fail(BC_ERR_DTYPE, "%s must be bf16 or f16", name);
    if (t.c % 8) return fail(BC_ERR_UNSUPPORTED, "%s: channels must be a multiple of 8", name);
    return BC_OK;
}

bc_status bc_policy_logit_grad(const float *d_reward, const uint8_t *d_mask, const float *d_prob,
                               void *d_grad, bc_tensor grad, void *stream)
{
    if (!d_reward || !d_mask || !d_prob || !d_grad)
        return fail(BC_ERR_NULL, "d_reward, d_mask, d_prob and d_grad are required");
    bc_status st;
    if ((st = check_grad_map(grad, "grad"))) return st;
    const double blocks = (double)grad.n * grad.h * grad.w;
    if (blocks > (double)(1 << 20)) return fail(BC_ERR_SHAPE, "more than 2^20 blocks");
    const size_t gb = tensor_bytes(grad), nb = (size_t)blocks;
    if (overlap(d_grad, gb, d_reward, nb * 4) || overlap(d_grad, gb, d_prob, nb * 4) ||
        overlap(d_grad, gb, d_mask, nb))
        return fail(BC_ERR_ALIAS, "d_grad overlaps an input");
    hipError_t e = bc::launch_logit_grad(d_reward, d_mask, d_prob, d_grad, (int)blocks, grad.c,
                                         grad.dtype == BC_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "logit gradient launch");
    return ok();
}

bc_status bc_grad_combine(const void *d_a, const void *d_b, const void *d_y, bc_tensor desc,
                          void *d_out, void *stream)
{
    if (!d_a || !d_out) return fail(BC_ERR_NULL, "d_a and d_out are required");
    bc_status st;
    if ((st = check_grad_map(desc, "desc"))) return st;
    const size_t bytes = tensor_bytes(desc);
    // out may equal a or b (elementwise, each element read before it is written), not
    // partially overlap them
    auto bad = [&](const void *p) { return p && p != d_out && overlap(d_out, bytes, p, bytes); };
    if (bad(d_a) || bad(d_b) || bad(d_y)) return fail(BC_ERR_ALIAS, "d_out partially overlaps an input");
    hipError_t e = bc::launch_grad_combine(d_a, d_b, d_y, d_out, (long long)bytes / 2,
                                           desc.dtype == BC_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "gradient combine launch");
    return ok();
}

// The forward layer of a backward call: input `in`, output gradient `gout` (shaped like
// the layer's output), geometry k x k, stride, pad = k / 2.
static bc_status train_geom(const bc_conv *geom, const bc_tensor &in, const bc_tensor &gout,
                            bc::LayerGeom &L)
{
    if (!geom) return fail(BC_ERR_NULL, "geometry is required");
    bc_status st;
    if ((st = check_grad_map(in, "in"))) return st;
    if ((st = check_grad_map(gout, "grad_out"))) return st;
    if (in.dtype != gout.dtype) return fail(BC_ERR_DTYPE, "in and grad_out dtypes differ");
    if (geom->kh != geom->kw || (geom->kh != 1 && geom->kh != 3))
        return fail(BC_ERR_UNSUPPORTED, "kernel must be 1x1 or 3x3");
    if (geom->stride != 1 && geom->stride != 2) return fail(BC_ERR_UNSUPPORTED, "stride must be 1 or 2");
    if (geom->pad != geom->kh / 2) return fail(BC_ERR_UNSUPPORTED, "pad must be k / 2");
    if (gout.n != in.n || gout.h * geom->stride != in.h || gout.w * geom->stride != in.w)
        return fail(BC_ERR_SHAPE, "grad_out must be the layer's output: [n][h/s][w/s][cout] with h, w "
                                  "multiples of the stride");
    if (gout.c % 64) return fail(BC_ERR_UNSUPPORTED, "output channels must be a multiple of 64");
    L.n = in.n; L.cin = in.c; L.hin = in.h; L.win = in.w;
    L.cout = gout.c; L.hout = gout.h; L.wout = gout.w;
    L.kh = geom->kh; L.kw = geom->kw; L.stride = geom->stride; L.pad = geom->pad;
    L.gh = L.gw = 1; L.bh = gout.h; L.bw = gout.w; L.total_blocks = in.n;
    L.idx = nullptr; L.count = nullptr;
    if (tensor_bytes(in) >= 2147483392u || tensor_bytes(gout) >= 2147483392u)
        return fail(BC_ERR_UNSUPPORTED, "tensors must be below 2 GiB");
    return BC_OK;
}

bc_status bc_conv2d_input_grad(const bc_conv *geom, const void *d_grad_out, bc_tensor grad_out,
                               const void *d_w, const void *d_accum, void *d_grad_in,
                               bc_tensor grad_in, void *stream)
{
    if (!d_grad_out || !d_w || !d_grad_in)
        return fail(BC_ERR_NULL, "d_grad_out, d_w and d_grad_in are required");
    bc::LayerGeom L;
    bc_status st = train_geom(geom, grad_in, grad_out, L);
    if (st) return st;
    if (grad_in.c % 64) return fail(BC_ERR_UNSUPPORTED, "input channels must be a multiple of 64");
    if (grad_in.h % 8 && grad_in.h > 8) return fail(BC_ERR_UNSUPPORTED, "input height must be <= 8 or a multiple of 8");
    if (grad_in.w % 8 && grad_in.w > 8) return fail(BC_ERR_UNSUPPORTED, "input width must be <= 8 or a multiple of 8");
    const size_t ib = tensor_bytes(grad_in), ob = tensor_bytes(grad_out);
    const size_t wb = (size_t)grad_out.c * geom->kh * geom->kw * grad_in.c * 2;
    if (overlap(d_grad_in, ib, d_grad_out, ob) || overlap(d_grad_in, ib, d_w, wb) ||
        overlap(d_grad_in, ib, d_accum, ib))
        return fail(BC_ERR_ALIAS, "d_grad_in overlaps an input");
    const char *why = "";
    hipError_t e = bc::launch_conv_input_grad(
        (const uint16_t *)d_grad_out, (const uint16_t *)d_w, (const uint16_t *)d_accum,
        (uint16_t *)d_grad_in, L, grad_in.dtype == BC_BF16 ? bc::Half16::BF16 : bc::Half16::F16,
        (hipStream_t)stream, &why);
    if (e != hipSuccess) return conv_fail(e, why, "input gradient launch");
    return ok();
}

bc_status bc_conv2d_weight_grad(const bc_conv *geom, const void *d_in, bc_tensor in,
                                const void *d_grad_out, bc_tensor grad_out, float *d_dw,
                                float *d_db, void *stream)
{
    if (!d_in || !d_grad_out || !d_dw) return fail(BC_ERR_NULL, "d_in, d_grad_out and d_dw are required");
    bc::LayerGeom L;
    bc_status st = train_geom(geom, in, grad_out, L);
    if (st) return st;
    const double wgs = (double)(grad_out.c / 64) * ((in.c + 63) / 64) * geom->kh * geom->kw *
                       std::ceil((double)in.n * grad_out.h * grad_out.w / 1024.0);
    if (wgs >= 4194304.0) return fail(BC_ERR_UNSUPPORTED, "too many pixels for one call");
    const size_t dwb = (size_t)grad_out.c * geom->kh * geom->kw * in.c * 4;
    if (overlap(d_dw, dwb, d_in, tensor_bytes(in)) || overlap(d_dw, dwb, d_grad_out, tensor_bytes(grad_out)) ||
        overlap(d_db, (size_t)grad_out.c * 4, d_dw, dwb))
        return fail(BC_ERR_ALIAS, "gradient outputs overlap each other or an input");
    hipError_t e = bc::launch_conv_weight_grad((const uint16_t *)d_in, (const uint16_t *)d_grad_out,
                                               d_dw, d_db, L, in.dtype == BC_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "weight gradient launch");
    return ok();
}

bc_status bc_rmsprop_step(float *d_w, float *d_v, float *d_grad, int64_t count, float lr,
                          float alpha, float eps, float weight_decay, void *d_w16, int32_t dtype,
                          void *stream)
{
    if (!d_w || !d_v || !d_grad) return fail(BC_ERR_NULL, "d_w, d_v and d_grad are required");
    if (count <= 0 || count > ((int64_t)1 << 31)) return fail(BC_ERR_SHAPE, "count outside 1..2^31");
    if (d_w16 && dtype != BC_BF16 && dtype != BC_F16) return fail(BC_ERR_DTYPE, "the copy must be bf16 or f16");
    const size_t b = (size_t)count * 4;
    if (overlap(d_w, b, d_v, b) || overlap(d_w, b, d_grad, b) || overlap(d_v, b, d_grad, b) ||
        overlap(d_w16, (size_t)count * 2, d_w, b) || overlap(d_w16, (size_t)count * 2, d_v, b) ||
        overlap(d_w16, (size_t)count * 2, d_grad, b))
        return fail(BC_ERR_ALIAS, "the optimiser's buffers overlap");
    hipError_t e = bc::launch_rmsprop(d_w, d_v, d_grad, (long long)count, lr, alpha, eps, weight_decay,
                                      d_w16, dtype == BC_BF16, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "rmsprop launch");
    return ok();
}

bc_status bc_rmsprop_step_many(const bc_param *params, int32_t n, float lr, float alpha, float eps,
                               float weight_decay, int32_t dtype, void *stream)
{
    if (!params) return fail(BC_ERR_NULL, "params is required");
    if (n < 1 || n > bc::kMaxParams) return fail(BC_ERR_SHAPE, "n outside 1..%d", bc::kMaxParams);
    bc::RmspropMany m{};
    m.n = n;
    bool any16 = false;
    long long blocks = 0;
    for (int t = 0; t < n; ++t) {
        const bc_param &p = params[t];
        if (!p.w || !p.v || !p.grad) return fail(BC_ERR_NULL, "params[%d]: w, v and grad are required", t);
        if (p.count <= 0 || p.count > ((int64_t)1 << 31)) return fail(BC_ERR_SHAPE, "params[%d]: count outside 1..2^31", t);
        any16 = any16 || p.w16;
        m.w[t] = p.w;
        m.v[t] = p.v;
        m.grad[t] = p.grad;
        m.w16[t] = (uint16_t *)p.w16;
        m.count[t] = p.count;
        m.first[t] = (int)blocks;
        blocks += (p.count + 255) / 256;
    }
    m.first[n] = (int)blocks;
    if (any16 && dtype != BC_BF16 && dtype != BC_F16) return fail(BC_ERR_DTYPE, "the copies must be bf16 or f16");
    // every buffer of every tensor against every other
    struct Span { const void *p; size_t b; };
    std::vector<Span> spans;
    for (int t = 0; t < n; ++t) {
        const size_t b = (size_t)params[t].count * 4;
        spans.push_back({params[t].w, b});
        spans.push_back({params[t].v, b});
        spans.push_back({params[t].grad, b});
        if (params[t].w16) spans.push_back({params[t].w16, (size_t)params[t].count * 2});
    }
    // sorted by start address, any overlap shows between neighbours
    std::sort(spans.begin(), spans.end(),
              [](const Span &x, const Span &y) { return (uintptr_t)x.p < (uintptr_t)y.p; });
    for (size_t i = 0; i + 1 < spans.size(); ++i)
        if (overlap(spans[i].p, spans[i].b, spans[i + 1].p, spans[i + 1].b))
            return fail(BC_ERR_ALIAS, "the optimiser's buffers overlap");
    hipError_t e = bc::launch_rmsprop_many(m, lr, alpha, eps, weight_decay, dtype == BC_BF16,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "rmsprop launch");
    return ok();
}

bc_status bc_block_rewards(const float *d_ig, const uint8_t *d_mask, const float *d_prob,
                           int32_t n, bc_grid g, float tau, float gamma, float mu, float *d_mavg,
                           float *d_reward, float *d_cost, float *d_loss, void *stream)
{
    if (!d_ig || !d_mask || !d_mavg || !d_reward)
        return fail(BC_ERR_NULL, "d_ig, d_mask, d_mavg and d_reward are required");
    if (d_loss && !d_prob) return fail(BC_ERR_NULL, "the loss needs d_prob");
    if (n <= 0 || g.grid_h <= 0 || g.grid_w <= 0)
        return fail(BC_ERR_SHAPE, "n and grid must be positive");
    const double total = (double)n * g.grid_h * g.grid_w;
    if (total > (double)(1 << 20)) return fail(BC_ERR_SHAPE, "more than 2^20 blocks");
    const size_t nb = (size_t)total;
    const void *outs[4] = {d_mavg, d_reward, d_cost, d_loss};
    const size_t outb[4] = {(size_t)n * 4, nb * 4, (size_t)n * 4, (size_t)n * 4};
    const void *ins[3] = {d_ig, d_mask, d_prob};
    const size_t inb[3] = {nb * 4, nb, nb * 4};
    for (int i = 0; i < 4; ++i) {
        for (int j = 0; j < 3; ++j)
            if (i > 0 && overlap(outs[i], outb[i], ins[j], inb[j]))   // d_mavg is in/out
                return fail(BC_ERR_ALIAS, "an output overlaps an input");
        for (int j = i + 1; j < 4; ++j)
            if (overlap(outs[i], outb[i], outs[j], outb[j]))
                return fail(BC_ERR_ALIAS, "outputs overlap each other");
    }
    for (int j = 0; j < 3; ++j)
        if (overlap(d_mavg, (size_t)n * 4, ins[j], inb[j]))
            return fail(BC_ERR_ALIAS, "d_mavg overlaps an input");
    hipError_t e = bc::launch_block_rewards(d_ig, d_mask, d_prob, n, g.grid_h * g.grid_w, tau, gamma,
                                            mu, d_mavg, d_reward, d_cost, d_loss, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "rewards launch");
    return ok();
}

}  // extern "C"
