// C-ABI entry points of libhatq: host-side validation and launch orchestration.
// Every argument check runs before the first HIP call, so invalid calls launch
// nothing, touch no output and need no GPU.
#include <hip/hip_runtime.h>

#include <cmath>
#include <vector>
#include <cstdint>
#include <cstring>

#include "../../include/hatq.h"
#include "hatq_launch.h"

namespace {

bool is_pow2(int v) { return v >= 1 && (v & (v - 1)) == 0; }

constexpr int32_t kMaxChannels = 1 << 16;   // per layer, in and out
constexpr int64_t kMaxElems = (int64_t)1 << 40;   // elements of one tensor

// a * b * c * d (all >= 1) without overflow, or -1 when above kMaxElems.
int64_t elems(int64_t a, int64_t b, int64_t c, int64_t d = 1) {
    int64_t v = 1;
    for (int64_t f : {a, b, c, d}) {
        if (f < 1 || v > kMaxElems / f) return -1;
        v *= f;
    }
    return v;
}
int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Transform orders the kernels implement: Sylvester blocks up to 128 and the
// Kronecker orders 192 = P_12 (x) H~_16 and 320 = P_20 (x) H~_16.
bool supported_order(int32_t b) { return (is_pow2(b) && b <= 128) || hatq::kron_q(b) != 0; }

int32_t check_desc(const hatq_conv_desc *d, int32_t form) {
    if (!d) return HATQ_EINVAL;
    if (form != HATQ_DH && form != HATQ_WH) return HATQ_EINVAL;
    if (d->cin <= 0 || d->cout <= 0 || d->k <= 0 || d->stride <= 0 || d->pad < 0 || d->out_pad < 0)
        return HATQ_EINVAL;
    // bounds that keep every derived size (k*k*cin_pad, cout_pad * k_stride) in range
    if (d->cin > kMaxChannels || d->cout > kMaxChannels || d->k > 64 || d->stride > 64 || d->pad > 64 ||
        d->out_pad > 64)
        return HATQ_EINVAL;
    if (!supported_order(d->hblock)) return HATQ_EINVAL;
    if (d->transposed != 0 && d->transposed != 1) return HATQ_EINVAL;
    if (d->transposed && d->out_pad >= d->stride) return HATQ_EINVAL;
    return HATQ_OK;
}

struct Dims {
    int32_t cin_p, cout_p, k_total, k_stride, pack_stride;
    bool rowrun;
};

// Row-run geometry: a regular convolution with a few input channels whose taps
// along one kernel row are k*cin_p <= 16 consecutive bytes of the NHWC input;
// its kernel contracts 16 bytes per kernel row (d' = 16*kh + kw*cin_p + ci).
bool rowrun_geometry(const hatq_conv_desc *d, int32_t cin_p) {
    return !d->transposed && cin_p <= 4 && d->k * cin_p <= 16 && d->k <= 8 && d->stride <= 2;
}

Dims dims_of(const hatq_conv_desc *d, int32_t form) {
    Dims r;
    r.cin_p = (int32_t)(form == HATQ_DH ? round_up(d->cin, d->hblock) : d->cin);
    r.cout_p = (int32_t)(form == HATQ_WH ? round_up(d->cout, d->hblock) : d->cout);
    r.k_total = d->k * d->k * r.cin_p;
    r.k_stride = (int32_t)round_up(r.k_total, 64);
    r.rowrun = rowrun_geometry(d, r.cin_p);
    r.pack_stride = r.rowrun ? (int32_t)round_up(16 * d->k, 64) : r.k_stride;
    return r;
}

int32_t out_hw(const hatq_conv_desc *d, int32_t h, int32_t w, int32_t *ho, int32_t *wo) {
    int64_t a, b;
    const int64_t H = h, Wd = w, p = d->pad, k = d->k, st = d->stride;
    if (d->transposed) {
        a = (H - 1) * st - 2 * p + k + d->out_pad;
        b = (Wd - 1) * st - 2 * p + k + d->out_pad;
    } else {
        if (H + 2 * p < k || Wd + 2 * p < k) return HATQ_EINVAL;
        a = (H + 2 * p - k) / st + 1;
        b = (Wd + 2 * p - k) / st + 1;
    }
    if (a <= 0 || b <= 0 || a > INT32_MAX || b > INT32_MAX) return HATQ_EINVAL;
    *ho = (int32_t)a;
    *wo = (int32_t)b;
    return HATQ_OK;
}

int32_t hip_status(hipError_t e) { return e == hipSuccess ? HATQ_OK : HATQ_EHIP; }

// An order b that spans several 64-channel blocks of the layer's tile of bn
// columns: a Kronecker order equal to the tile (192; 320 on the general
// kernel's 320-column tile, which the small-channel kernels lack), or the
// Sylvester order 128 on tiles of 128 or 256 columns (not on the
// small-channel gather kernel).
bool kron_tile(const hatq_weights *W, int b, int bn) {
    const bool small = W->cin_pad <= 4 && W->k_total <= 128;
    if (b == 128) return (bn == 128 || bn == 256) && (!small || rowrun_geometry(&W->d, W->cin_pad));
    return (b == 192 && bn == 192) || (b == 320 && bn == 320 && !small);
}

// Kernel geometry the conv kernels implement.
int32_t check_conv_supported(const hatq_weights *W) {
    const hatq_conv_desc &d = W->d;
    const bool small = W->cin_pad <= 4 && W->k_total <= 128;
    if (!small && W->cin_pad % 64 != 0) return HATQ_EUNSUPPORTED;
    if (W->cout_pad % 64 != 0) return HATQ_EUNSUPPORTED;
    const bool rowrun = rowrun_geometry(&d, W->cin_pad);
    if (!rowrun && d.k * d.k > hatq::kMaxTaps) return HATQ_EUNSUPPORTED;   // tap table
    if (d.transposed && (d.stride != 2 || small)) return HATQ_EUNSUPPORTED;
    if (d.k > 64 || d.pad > 64 || d.stride > 64) return HATQ_EUNSUPPORTED;
    // the WH restore runs inside one wave: the block must tile the wave's columns
    const int tiles[] = {64, 128, 192, 256, 320};
    bool fixed = false;
    for (int t : tiles) fixed |= (W->cout_pad == t);
    const int bn = fixed ? W->cout_pad : 64;
    // the WH restore runs inside one wave: a Sylvester block up to 64 that tiles
    // the columns, or a wider order on a tile that holds whole blocks of it
    // (kron_tile)
    if (W->form == HATQ_WH) {
        const int b = W->d.hblock;
        const bool ok = (is_pow2(b) && b <= 64 && bn % b == 0) || kron_tile(W, b, bn);
        if (!ok) return HATQ_EUNSUPPORTED;
    }
    return HATQ_OK;
}

int32_t check_weights(const hatq_weights *W) {
    if (!W) return HATQ_EINVAL;
    if (check_desc(&W->d, W->form) != HATQ_OK) return HATQ_EINVAL;
    const Dims dm = dims_of(&W->d, W->form);
    if (dm.cin_p != W->cin_pad || dm.cout_p != W->cout_pad || dm.k_total != W->k_total ||
        dm.k_stride != W->k_stride || dm.pack_stride != W->pack_stride)
        return HATQ_EINVAL;
    if (!W->wq || !W->w_scale || !W->bias || !W->wpack) return HATQ_EINVAL;
    if (!aligned(W->wq, 16) || !aligned(W->w_scale, 16) || !aligned(W->bias, 16) || !aligned(W->wpack, 16))
        return HATQ_EINVAL;
    return HATQ_OK;
}

// The chunk-major layouts: HATQ_XQ_C64 for the 5x5 stride-2 window kernel,
// HATQ_YQ_C64 for code outputs with whole 64-channel planes.
constexpr int32_t kConvFlags = HATQ_PAIRED | HATQ_XQ_C64 | HATQ_YQ_C64;
// order320: the launch applies an order-320 transform in its epilogue (the WH
// restore of a float or code output, or the next operand's), which runs on the
// general kernel's 320-column tile, not on the window kernel that reads
// chunk-major codes.
int32_t check_layouts(const hatq_weights *W, int32_t flags, bool codes_out, bool order320 = false) {
    const hatq_conv_desc &d = W->d;
    if ((flags & HATQ_YQ_C64) && !codes_out) return HATQ_EINVAL;
    if ((flags & HATQ_YQ_C64) && d.cout % 64 != 0) return HATQ_EUNSUPPORTED;
    if ((flags & HATQ_XQ_C64) &&
        (d.transposed || d.k != 5 || d.stride != 2 || W->cin_pad % 64 != 0 ||
         (W->cout_pad != 192 && W->cout_pad != 320) || order320))
        return HATQ_EUNSUPPORTED;
    return HATQ_OK;
}

// Whether a launch with a float or code output (not I32) transforms by the
// order 320 in its epilogue.
bool order320(const hatq_weights *W, int32_t next_hblock, bool next_used) {
    return (W->form == HATQ_WH && W->d.hblock == 320) || (next_used && next_hblock == 320);
}

int32_t check_next(const hatq_weights *W, int32_t next_hblock, const float *next_absmax) {
    if (!next_absmax) return HATQ_OK;
    if (!supported_order(next_hblock)) return HATQ_EINVAL;
    if (W->d.cout % next_hblock != 0) return HATQ_EUNSUPPORTED;
    const int tiles[] = {64, 128, 192, 256, 320};
    bool fixed = false;
    for (int t : tiles) fixed |= (W->cout_pad == t);
    const int bn = fixed ? W->cout_pad : 64;
    // the next operand's transform runs inside one wave: a Sylvester block up
    // to 64 that tiles the columns, or a wider order on a tile that holds whole
    // blocks of it (kron_tile)
    if (hatq::kron_q(next_hblock) || next_hblock == 128) {
        if (!kron_tile(W, next_hblock, bn)) return HATQ_EUNSUPPORTED;
    } else if (next_hblock > 64 || (bn % next_hblock != 0 && next_hblock > 1)) {
        return HATQ_EUNSUPPORTED;
    }
    if (!aligned(next_absmax, 4)) return HATQ_EINVAL;
    return HATQ_OK;
}

// Fill the tap table of one GEMM launch.  Regular convolution: one launch over
// the output grid, taps (kh, kw).  Transposed convolution with stride 2: one
// launch per output phase (ph, pw) over the points (i, j) with
// oh = 2i + ph; tap kh is used iff (oh + pad - kh) is even, and then reads input
// row i + (ph + pad - kh)/2 (gather form of the transposed convolution).
int32_t conv_launches(const hatq_weights *W, const int8_t *xq, const float *sx, int32_t n,
                      int32_t h, int32_t w, int32_t mode, void *y, int32_t next_hblock,
                      float *next_absmax, int32_t flags, hipStream_t st, const float *q_absmax = nullptr,
                      float *q_scale = nullptr, const int32_t *rq_table = nullptr,
                      const int32_t *zx = nullptr, const int32_t *tapsum = nullptr) {
    const hatq_conv_desc &d = W->d;
    int32_t ho, wo;
    if (out_hw(&d, h, w, &ho, &wo) != HATQ_OK) return HATQ_EINVAL;
    if (elems(n, h, w, W->cin_pad) < 0 || elems(n, ho, wo, W->cout_pad) < 0) return HATQ_EINVAL;
    hatq::ConvArgs a;
    std::memset(&a, 0, sizeof(a));
    a.xq = xq;
    a.wp = W->wpack;
    a.sx = sx;
    a.w_scale = W->w_scale;
    a.bias = W->bias;
    a.y = y;
    a.next_absmax = next_absmax;
    a.q_absmax = q_absmax;
    a.q_scale = q_scale;
    a.rq_table = rq_table;
    a.zx = zx;
    a.tapsum = tapsum;
    a.n = n;
    a.h = h;
    a.w = w;
    a.cin_p = W->cin_pad;
    a.ho = ho;
    a.wo = wo;
    a.k = d.k;
    a.k_total = W->k_total;
    a.pack_stride = W->pack_stride;
    a.rowrun = rowrun_geometry(&d, W->cin_pad);
    a.cout = d.cout;
    a.cout_pad = W->cout_pad;
    a.form = W->form;
    a.mode = mode;
    a.hblock = d.hblock;
    a.next_hblock = (next_absmax || mode >= HATQ_OUT_I8) ? next_hblock : 0;
    a.paired = (flags & HATQ_PAIRED) ? 1 : 0;
    a.xq_c64 = (flags & HATQ_XQ_C64) ? 1 : 0;
    a.yq_c64 = (flags & HATQ_YQ_C64) ? 1 : 0;
    const bool small = W->cin_pad <= 4 && W->k_total <= 128;
    if (!d.transposed) {
        a.gh = ho;
        a.gw = wo;
        a.sa = d.stride;
        a.bah = -d.pad;
        a.baw = -d.pad;
        a.so = 1;
        a.boh = 0;
        a.bow = 0;
        a.ntaps = d.k * d.k;
        for (int kh = 0; kh < d.k && d.k * d.k <= hatq::kMaxTaps; ++kh)   // (row-run needs no table)
            for (int kw = 0; kw < d.k; ++kw) {
                const int t = kh * d.k + kw;
                a.dh[t] = (int8_t)kh;
                a.dw[t] = (int8_t)kw;
                a.wtap[t] = (int16_t)t;
            }
        a.nksteps = small ? W->pack_stride / 64 : a.ntaps * (W->cin_pad / 64);
        a.M = (int64_t)n * a.gh * a.gw;
        return hip_status(hatq::launch_conv(a, true, st));
    }
    // transposed, stride 2: four phases
    bool first = true;
    for (int ph = 0; ph < 2; ++ph)
        for (int pw = 0; pw < 2; ++pw) {
            hatq::ConvArgs b = a;
            b.gh = (ho - ph + 1) / 2;
            b.gw = (wo - pw + 1) / 2;
            if (b.gh <= 0 || b.gw <= 0) continue;
            b.sa = 1;
            b.bah = 0;
            b.baw = 0;
            b.so = 2;
            b.boh = ph;
            b.bow = pw;
            int nt = 0;
            for (int kh = 0; kh < d.k; ++kh) {
                if (((ph + d.pad - kh) % 2 + 2) % 2) continue;
                for (int kw = 0; kw < d.k; ++kw) {
                    if (((pw + d.pad - kw) % 2 + 2) % 2) continue;
                    b.dh[nt] = (int8_t)((ph + d.pad - kh) / 2);
                    b.dw[nt] = (int8_t)((pw + d.pad - kw) / 2);
                    b.wtap[nt] = (int16_t)(kh * d.k + kw);
                    ++nt;
                }
            }
            b.ntaps = nt;
            b.nksteps = nt * (W->cin_pad / 64);
            b.M = (int64_t)n * b.gh * b.gw;
            if (nt == 0) continue;   // cannot happen for k >= 2
            // next_absmax is cleared by the first phase and accumulated by the rest
            if (hatq::launch_conv(b, first, st) != hipSuccess) return HATQ_EHIP;
            first = false;
        }
    return HATQ_OK;
}

}  // namespace

extern "C" {

const char *hatq_status_string(int32_t s) {
    switch (s) {
        case HATQ_OK: return "ok";
        case HATQ_EINVAL: return "invalid argument";
        case HATQ_EUNSUPPORTED: return "unsupported geometry";
        case HATQ_EWORKSPACE: return "workspace too small";
        case HATQ_EHIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

int32_t hatq_conv_out_hw(const hatq_conv_desc *d, int32_t h, int32_t w, int32_t *ho, int32_t *wo) {
    if (!d || !ho || !wo || h <= 0 || w <= 0) return HATQ_EINVAL;
    if (check_desc(d, HATQ_DH) != HATQ_OK) return HATQ_EINVAL;
    return out_hw(d, h, w, ho, wo);
}

size_t hatq_weights_bytes(const hatq_conv_desc *d, int32_t form) {
    if (check_desc(d, form) != HATQ_OK) return 0;
    const Dims dm = dims_of(d, form);
    return align256((size_t)dm.cout_p * dm.k_stride) + 2 * align256((size_t)dm.cout_p * 4) +
           align256((size_t)dm.cout_p * dm.pack_stride);
}

int32_t hatq_prepare_weights(const hatq_conv_desc *d, int32_t form, const float *w, const float *bias,
                             void *dst, size_t dst_bytes, hatq_weights *out, void *stream) {
    if (check_desc(d, form) != HATQ_OK || !w || !dst || !out) return HATQ_EINVAL;
    if (form == HATQ_DH && d->cin % d->hblock) return HATQ_EUNSUPPORTED;
    if (form == HATQ_WH && d->cout % d->hblock) return HATQ_EUNSUPPORTED;
    if (!aligned(dst, 256) || !aligned(w, 4) || (bias && !aligned(bias, 4))) return HATQ_EINVAL;
    const size_t need = hatq_weights_bytes(d, form);
    if (dst_bytes < need) return HATQ_EWORKSPACE;
    const Dims dm = dims_of(d, form);
    hatq_weights W;
    W.d = *d;
    W.form = form;
    W.cin_pad = dm.cin_p;
    W.cout_pad = dm.cout_p;
    W.k_total = dm.k_total;
    W.k_stride = dm.k_stride;
    int8_t *base = static_cast<int8_t *>(dst);
    W.wq = base;
    W.w_scale = reinterpret_cast<float *>(base + align256((size_t)dm.cout_p * dm.k_stride));
    W.bias = reinterpret_cast<float *>(reinterpret_cast<int8_t *>(W.w_scale) + align256((size_t)dm.cout_p * 4));
    W.wpack = reinterpret_cast<int8_t *>(W.bias) + align256((size_t)dm.cout_p * 4);
    W.pack_stride = dm.pack_stride;
    hatq::PrepArgs a;
    a.w = w;
    a.bias = bias;
    a.wq = W.wq;
    a.w_scale = W.w_scale;
    a.w_bias = W.bias;
    a.cin = d->cin;
    a.cout = d->cout;
    a.k = d->k;
    a.transposed = d->transposed;
    a.hblock = d->hblock;
    a.form = form;
    a.cin_p = dm.cin_p;
    a.cout_p = dm.cout_p;
    a.k_total = dm.k_total;
    a.k_stride = dm.k_stride;
    a.wpack = W.wpack;
    a.pack_stride = dm.pack_stride;
    a.rowrun = dm.rowrun;
    const int32_t st = hip_status(hatq::launch_prepare(a, static_cast<hipStream_t>(stream)));
    if (st == HATQ_OK) *out = W;
    return st;
}

int32_t hatq_pack_weights(const hatq_weights *W, void *stream) {
    const int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    hatq::PrepArgs a;
    std::memset(&a, 0, sizeof(a));
    a.wq = W->wq;
    a.wpack = W->wpack;
    a.k = W->d.k;
    a.cin_p = W->cin_pad;
    a.cout_p = W->cout_pad;
    a.k_total = W->k_total;
    a.k_stride = W->k_stride;
    a.pack_stride = W->pack_stride;
    a.rowrun = rowrun_geometry(&W->d, W->cin_pad);
    return hip_status(hatq::launch_pack(a, static_cast<hipStream_t>(stream)));
}

int32_t hatq_export_weights(const hatq_weights *W, int8_t *wq, float *w_scale, float *bias, void *stream) {
    const int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (wq && hipMemcpy2DAsync(wq, (size_t)W->k_total, W->wq, (size_t)W->k_stride, (size_t)W->k_total,
                               (size_t)W->cout_pad, hipMemcpyDefault, st) != hipSuccess)
        return HATQ_EHIP;
    const size_t cb = (size_t)W->cout_pad * sizeof(float);
    if (w_scale && hipMemcpyAsync(w_scale, W->w_scale, cb, hipMemcpyDefault, st) != hipSuccess) return HATQ_EHIP;
    if (bias && hipMemcpyAsync(bias, W->bias, cb, hipMemcpyDefault, st) != hipSuccess) return HATQ_EHIP;
    return HATQ_OK;
}

size_t hatq_fwht_quant_ws_bytes(int32_t n) { return n > 0 ? align256((size_t)n * 4 * hatq::kAbsSlots) : 0; }

int32_t hatq_fwht_quant_act(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                            const float *absmax, int8_t *xq, float *act_scale, void *ws, size_t ws_bytes,
                            void *stream) {
    if (!x || !xq || !act_scale || n <= 0 || h <= 0 || w <= 0 || c <= 0) return HATQ_EINVAL;
    if (!supported_order(hblock)) return HATQ_EINVAL;
    if (c % hblock) return HATQ_EUNSUPPORTED;
    if (!aligned(x, 16) || !aligned(xq, 4) || !aligned(act_scale, 4)) return HATQ_EINVAL;
    if (absmax && !aligned(absmax, 4)) return HATQ_EINVAL;
    if (elems(n, h, w, c) < 0) return HATQ_EINVAL;
    if (!absmax) {
        if (!ws) return HATQ_EINVAL;
        if (ws_bytes < hatq_fwht_quant_ws_bytes(n) || !aligned(ws, 4)) return HATQ_EWORKSPACE;
    }
    const int64_t E = (int64_t)h * w * c;
    return hip_status(hatq::launch_act_quant(x, n, E, hblock, absmax, static_cast<float *>(ws), xq,
                                             act_scale, static_cast<hipStream_t>(stream)));
}

int32_t hatq_fwht_quant_act_c64(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                                const float *absmax, int8_t *xq, float *act_scale, void *ws, size_t ws_bytes,
                                void *stream) {
    if (!x || !xq || !act_scale || n <= 0 || h <= 0 || w <= 0 || c <= 0) return HATQ_EINVAL;
    if (!supported_order(hblock)) return HATQ_EINVAL;
    if (c % 64 != 0 || hblock > 64 || (hblock & (hblock - 1)) != 0) return HATQ_EUNSUPPORTED;
    if (!aligned(x, 16) || !aligned(xq, 16) || !aligned(act_scale, 4)) return HATQ_EINVAL;
    if (absmax && !aligned(absmax, 4)) return HATQ_EINVAL;
    if (elems(n, h, w, c) < 0) return HATQ_EINVAL;
    if (!absmax) {
        if (!ws) return HATQ_EINVAL;
        if (ws_bytes < hatq_fwht_quant_ws_bytes(n) || !aligned(ws, 4)) return HATQ_EWORKSPACE;
    }
    const int64_t E = (int64_t)h * w * c;
    return hip_status(hatq::launch_act_quant(x, n, E, hblock, absmax, static_cast<float *>(ws), xq, act_scale,
                                             static_cast<hipStream_t>(stream), c));
}

int32_t hatq_fwht_quant_act_noalloc(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                                    int8_t *xq, float *act_scale, void *stream) {
    static_assert(HATQ_NOALLOC_MAX_SAMPLES == hatq::kNoAllocMaxSamples, "one limit");
    if (!x || !xq || !act_scale || n <= 0 || h <= 0 || w <= 0 || c <= 0) return HATQ_EINVAL;
    if (!supported_order(hblock)) return HATQ_EINVAL;
    if (c % hblock) return HATQ_EUNSUPPORTED;
    if (!aligned(x, 16) || !aligned(xq, 4) || !aligned(act_scale, 4)) return HATQ_EINVAL;
    if (n > HATQ_NOALLOC_MAX_SAMPLES) return HATQ_EUNSUPPORTED;
    if (elems(n, h, w, c) < 0) return HATQ_EINVAL;
    const int64_t E = (int64_t)h * w * c;
    return hip_status(hatq::launch_act_quant_noalloc(x, n, E, hblock, xq, act_scale, static_cast<hipStream_t>(stream)));
}

namespace {

// The requantizing epilogue (I8 output): dynamic scale from next_absmax, or the
// static scale in next_scale.
int32_t requant(const hatq_weights *W, const int8_t *xq, const float *act_scale, int32_t n, int32_t h, int32_t w,
                int32_t next_hblock, const float *next_absmax, float *next_scale, int8_t *yq, int32_t flags,
                void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (!xq || !act_scale || !next_scale || !yq || n <= 0 || h <= 0 || w <= 0) return HATQ_EINVAL;
    if (flags & ~kConvFlags) return HATQ_EINVAL;
    if (!aligned(xq, 16) || !aligned(yq, (flags & HATQ_YQ_C64) ? 16 : 4) || !aligned(act_scale, 4) ||
        !aligned(next_scale, 4))
        return HATQ_EINVAL;
    if (next_absmax && !aligned(next_absmax, 4)) return HATQ_EINVAL;
    if ((s = check_conv_supported(W)) != HATQ_OK) return s;
    if ((s = check_layouts(W, flags, true, order320(W, next_hblock, true))) != HATQ_OK) return s;
    // the transform and the code layout follow the next operand's blocks
    const float *probe = next_absmax ? next_absmax : next_scale;
    if ((s = check_next(W, next_hblock, probe)) != HATQ_OK) return s;
    if (W->d.cout % 4) return HATQ_EUNSUPPORTED;
    int32_t ho, wo;
    if (out_hw(&W->d, h, w, &ho, &wo) != HATQ_OK) return HATQ_EINVAL;
    return conv_launches(W, xq, act_scale, n, h, w, HATQ_OUT_I8, yq, next_hblock, nullptr, flags,
                         static_cast<hipStream_t>(stream), next_absmax, next_scale);
}

}  // namespace

int32_t hatq_conv_int8(const hatq_weights *W, const int8_t *xq, const float *act_scale, int32_t n, int32_t h,
                       int32_t w, int32_t out_mode, const float *out_scale, void *y, int32_t next_hblock,
                       float *next_absmax, int32_t flags, void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (!xq || !act_scale || n <= 0 || h <= 0 || w <= 0) return HATQ_EINVAL;
    if (flags & ~kConvFlags) return HATQ_EINVAL;
    if (out_mode == HATQ_OUT_I8) {
        // requantization with a static per-sample scale (read, never written)
        if (!out_scale || !y || next_absmax) return HATQ_EINVAL;
        return requant(W, xq, act_scale, n, h, w, next_hblock, nullptr, const_cast<float *>(out_scale),
                       static_cast<int8_t *>(y), flags, stream);
    }
    if (out_mode != HATQ_OUT_I32 && out_mode != HATQ_OUT_F32) return HATQ_EINVAL;
    if (out_scale) return HATQ_EINVAL;
    if (out_mode == HATQ_OUT_I32 && next_absmax) return HATQ_EINVAL;
    // y may be NULL only when the call is for next_absmax alone
    if (!y && !(out_mode == HATQ_OUT_F32 && next_absmax)) return HATQ_EINVAL;
    if (!aligned(xq, 16) || (y && !aligned(y, 16)) || !aligned(act_scale, 4)) return HATQ_EINVAL;
    if ((s = check_conv_supported(W)) != HATQ_OK) return s;
    if ((s = check_layouts(W, flags, false,
                           out_mode == HATQ_OUT_F32 && order320(W, next_hblock, next_absmax != nullptr))) !=
        HATQ_OK)
        return s;
    if ((s = check_next(W, next_hblock, next_absmax)) != HATQ_OK) return s;
    int32_t ho, wo;
    if (out_hw(&W->d, h, w, &ho, &wo) != HATQ_OK) return HATQ_EINVAL;
    return conv_launches(W, xq, act_scale, n, h, w, out_mode, y, next_hblock, next_absmax, flags,
                         static_cast<hipStream_t>(stream));
}

int32_t hatq_conv_int8_requant(const hatq_weights *W, const int8_t *xq, const float *act_scale, int32_t n,
                               int32_t h, int32_t w, int32_t next_hblock, const float *next_absmax,
                               float *next_scale, int8_t *yq, int32_t flags, void *stream) {
    return requant(W, xq, act_scale, n, h, w, next_hblock, next_absmax, next_scale, yq, flags, stream);
}

size_t hatq_fwht_quant_affine_ws_bytes(int32_t n) { return n > 0 ? align256((size_t)n * 8) : 0; }

int32_t hatq_fwht_quant_act_affine(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                                   int8_t *xq, float *act_scale, int32_t *act_zero, void *ws, size_t ws_bytes,
                                   void *stream) {
    if (!x || !xq || !act_scale || !act_zero || !ws || n <= 0 || n > 65535 || h <= 0 || w <= 0 || c <= 0)
        return HATQ_EINVAL;
    if (!supported_order(hblock)) return HATQ_EINVAL;
    if (!aligned(x, 16) || !aligned(xq, 4) || !aligned(act_scale, 4) || !aligned(act_zero, 4) || !aligned(ws, 4))
        return HATQ_EINVAL;
    if (ws_bytes < (size_t)n * 8) return HATQ_EWORKSPACE;
    if (elems(n, h, w, c) < 0) return HATQ_EINVAL;
    const int64_t E = (int64_t)h * w * c;
    if (c % hblock != 0 || E % 4 != 0) return HATQ_EUNSUPPORTED;
    return hip_status(hatq::launch_act_quant_affine(x, n, E, hblock, static_cast<float *>(ws), xq, act_scale,
                                                    act_zero, static_cast<hipStream_t>(stream)));
}

size_t hatq_tapsum_len(const hatq_weights *W) {
    if (check_weights(W) != HATQ_OK) return 0;
    return ((size_t)W->d.k * W->d.k + 1) * W->cout_pad;
}

int32_t hatq_weight_tapsums(const hatq_weights *W, int32_t *tapsum, void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (!tapsum || !aligned(tapsum, 16)) return HATQ_EINVAL;
    if (W->d.k * W->d.k > 256) return HATQ_EUNSUPPORTED;   // one thread per tap
    hatq::PrepArgs a;
    std::memset(&a, 0, sizeof(a));
    a.wq = W->wq;
    a.k = W->d.k;
    a.cin_p = W->cin_pad;
    a.cout_p = W->cout_pad;
    a.k_total = W->k_total;
    a.k_stride = W->k_stride;
    return hip_status(hatq::launch_tapsums(a, tapsum, static_cast<hipStream_t>(stream)));
}

int32_t hatq_conv_int8_affine(const hatq_weights *W, const int8_t *xq, const float *act_scale,
                              const int32_t *act_zero, const int32_t *tapsum, int32_t n, int32_t h, int32_t w,
                              int32_t out_mode, void *y, void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (!xq || !act_scale || !act_zero || !tapsum || !y || n <= 0 || h <= 0 || w <= 0) return HATQ_EINVAL;
    if (out_mode != HATQ_OUT_I32 && out_mode != HATQ_OUT_F32) return HATQ_EINVAL;
    if (!aligned(xq, 16) || !aligned(y, 16) || !aligned(act_scale, 4) || !aligned(act_zero, 4) ||
        !aligned(tapsum, 16))
        return HATQ_EINVAL;
    if ((s = check_conv_supported(W)) != HATQ_OK) return s;
    // (the zero-point correction's wide-order variant covers the Kronecker orders)
    if (W->form == HATQ_WH && W->d.hblock == 128) return HATQ_EUNSUPPORTED;
    int32_t ho, wo;
    if (out_hw(&W->d, h, w, &ho, &wo) != HATQ_OK) return HATQ_EINVAL;
    return conv_launches(W, xq, act_scale, n, h, w, out_mode, y, 0, nullptr, 0, static_cast<hipStream_t>(stream),
                         nullptr, nullptr, nullptr, act_zero, tapsum);
}

size_t hatq_int_table_len(const hatq_weights *W) {
    if (check_weights(W) != HATQ_OK) return 0;
    return 2 * (size_t)W->cout_pad + 1;
}

int32_t hatq_int_transition_params(const hatq_weights *W, float s_x, float s_y, int32_t next_hblock,
                                   int32_t *table, void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (!table || !aligned(table, 16)) return HATQ_EINVAL;
    if (!(s_x > 0.0f) || !(s_y > 0.0f) || !std::isfinite(s_x) || !std::isfinite(s_y)) return HATQ_EINVAL;
    if (W->form == HATQ_WH && W->d.hblock == 128) return HATQ_EUNSUPPORTED;   // as the transition itself
    if (!((is_pow2(next_hblock) && next_hblock <= 64) || hatq::kron_q(next_hblock) != 0)) return HATQ_EINVAL;
    const bool dh = W->form == HATQ_DH;
    hatq::IntParamArgs a;
    a.w_scale = W->w_scale;
    a.bias = W->bias;
    a.table = table;
    a.s_x = s_x;
    a.s_y = s_y;
    a.cout_p = W->cout_pad;
    a.beta_in = dh ? W->d.hblock : 1;
    a.beta_out = dh ? 1 : W->d.hblock;
    a.K = W->d.k * W->d.k * W->cin_pad;
    a.gain = a.beta_out * next_hblock;
    return hip_status(hatq::launch_int_params(a, static_cast<hipStream_t>(stream)));
}

int32_t hatq_conv_int8_int_transition(const hatq_weights *W, const int8_t *xq, int32_t n, int32_t h, int32_t w,
                                      int32_t next_hblock, const int32_t *table, int8_t *yq, int32_t flags,
                                      void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (!xq || !table || !yq || n <= 0 || h <= 0 || w <= 0) return HATQ_EINVAL;
    if (flags & ~kConvFlags) return HATQ_EINVAL;
    if (!aligned(xq, 16) || !aligned(yq, (flags & HATQ_YQ_C64) ? 16 : 4) || !aligned(table, 16)) return HATQ_EINVAL;
    if ((s = check_conv_supported(W)) != HATQ_OK) return s;
    if ((s = check_layouts(W, flags, true, order320(W, next_hblock, true))) != HATQ_OK) return s;
    if ((s = check_next(W, next_hblock, reinterpret_cast<const float *>(table))) != HATQ_OK) return s;
    // (the integer epilogue takes the Sylvester order 128 on neither side)
    if (next_hblock == 128 || (W->form == HATQ_WH && W->d.hblock == 128)) return HATQ_EUNSUPPORTED;
    if (W->d.cout % 4) return HATQ_EUNSUPPORTED;
    int32_t ho, wo;
    if (out_hw(&W->d, h, w, &ho, &wo) != HATQ_OK) return HATQ_EINVAL;
    return conv_launches(W, xq, nullptr, n, h, w, hatq::kModeIntTransition, yq, next_hblock, nullptr, flags,
                         static_cast<hipStream_t>(stream), nullptr, nullptr, table);
}

int32_t hatq_range_expansion(const float *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t hblock,
                             float *amax, int32_t *flags, int32_t *count, void *stream) {
    if (!x || !amax || n <= 0 || n > 65535 || h <= 0 || w <= 0 || c <= 0) return HATQ_EINVAL;
    if (!supported_order(hblock)) return HATQ_EINVAL;
    if (!aligned(x, 16) || !aligned(amax, 4)) return HATQ_EINVAL;
    if ((flags && !aligned(flags, 4)) || (count && !aligned(count, 4))) return HATQ_EINVAL;
    if (elems(n, h, w, c) < 0) return HATQ_EINVAL;
    const int64_t P = (int64_t)h * w;
    // Kronecker orders: whole blocks and float4-aligned samples only
    if (!is_pow2(hblock) && (c % hblock != 0 || (P * c) % 4 != 0)) return HATQ_EUNSUPPORTED;
    return hip_status(hatq::launch_range_expansion(x, n, P, c, hblock, amax, flags, count,
                                                   static_cast<hipStream_t>(stream)));
}

int32_t hatq_select_form(int64_t expansions, int64_t images, double tau, int32_t *form) {
    if (!form || images <= 0 || expansions < 0 || expansions > images || !std::isfinite(tau)) return HATQ_EINVAL;
    const double p = (double)expansions / (double)images;
    *form = p > tau ? HATQ_WH : HATQ_DH;
    return HATQ_OK;
}

int32_t hatq_hadamard_order(int32_t c) {
    constexpr int kMax = 4096;
    if (c < 1 || c > kMax) return 0;
    // orders with a construction: 1, 2, Paley-I q + 1 (q = 3 mod 4) and
    // Paley-II 2(q + 1) (q = 1 mod 4) for odd prime powers q, and products
    static const std::vector<bool> built = [] {
        std::vector<bool> ok(kMax + 1, false);
        auto prime_power = [](int q) {
            int p = 2;
            while (q % p) ++p;
            while (q % p == 0) q /= p;
            return q == 1;
        };
        ok[1] = ok[2] = true;
        for (int q = 3; q < kMax; q += 2) {
            if (!prime_power(q)) continue;
            if (q % 4 == 3 && q + 1 <= kMax) ok[q + 1] = true;
            if (q % 4 == 1 && 2 * (q + 1) <= kMax) ok[2 * (q + 1)] = true;
        }
        for (int m = 4; m <= kMax; ++m)
            for (int a = 2; a * a <= m && !ok[m]; ++a)
                if (m % a == 0 && ok[a] && ok[m / a]) ok[m] = true;
        return ok;
    }();
    for (int m = 4 * ((c + 3) / 4); m <= kMax; m += 4)
        if (built[m]) return m;
    return 0;
}

size_t hatq_layer_ws_bytes(const hatq_weights *W, int32_t n, int32_t h, int32_t w) {
    if (check_weights(W) != HATQ_OK || n <= 0 || h <= 0 || w <= 0) return 0;
    if (elems(n, h, w, W->cin_pad) < 0) return 0;
    const size_t codes = (size_t)n * h * w * W->cin_pad;
    return align256(codes) + align256((size_t)n * 4) + hatq_fwht_quant_ws_bytes(n);
}

int32_t hatq_layer_forward(const hatq_weights *W, int32_t form, const float *x, int32_t n, int32_t h, int32_t w,
                           const float *x_absmax, float *y, float *act_scale, int32_t next_hblock,
                           float *next_absmax, void *ws, size_t ws_bytes, void *stream) {
    int32_t s = check_weights(W);
    if (s != HATQ_OK) return s;
    if (form != W->form) return HATQ_EINVAL;
    if (!x || !y || !ws || n <= 0 || h <= 0 || w <= 0) return HATQ_EINVAL;
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(ws, 256)) return HATQ_EINVAL;
    if (act_scale && !aligned(act_scale, 4)) return HATQ_EINVAL;
    if (x_absmax && !aligned(x_absmax, 4)) return HATQ_EINVAL;
    if ((s = check_conv_supported(W)) != HATQ_OK) return s;
    if ((s = check_next(W, next_hblock, next_absmax)) != HATQ_OK) return s;
    const int hb_act = form == HATQ_DH ? W->d.hblock : 1;
    if (W->cin_pad != W->d.cin) return HATQ_EUNSUPPORTED;   // activation padding not supported
    if (W->d.cin % hb_act) return HATQ_EUNSUPPORTED;
    int32_t ho, wo;
    if (out_hw(&W->d, h, w, &ho, &wo) != HATQ_OK) return HATQ_EINVAL;
    if (elems(n, h, w, W->cin_pad) < 0 || elems(n, ho, wo, W->cout_pad) < 0) return HATQ_EINVAL;
    const size_t need = hatq_layer_ws_bytes(W, n, h, w);
    if (ws_bytes < need) return HATQ_EWORKSPACE;
    int8_t *xq = static_cast<int8_t *>(ws);
    float *ws_sx = reinterpret_cast<float *>(xq + align256((size_t)n * h * w * W->cin_pad));
    float *amax = reinterpret_cast<float *>(reinterpret_cast<int8_t *>(ws_sx) + align256((size_t)n * 4));
    float *sx = act_scale ? act_scale : ws_sx;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int64_t E = (int64_t)h * w * W->d.cin;
    if (hatq::launch_act_quant(x, n, E, hb_act, x_absmax, amax, xq, sx, st) != hipSuccess) return HATQ_EHIP;
    return conv_launches(W, xq, sx, n, h, w, HATQ_OUT_F32, y, next_hblock, next_absmax, 0, st);
}

}  // extern "C"
