// Argument validation of the C ABI under AddressSanitizer and UndefinedBehavior-
// Sanitizer: every call below must be rejected on the host (fake, never
// dereferenced device pointers; extreme sizes that overflow naive products).
#include <cstdint>
#include <cstdio>

#include "../../include/hatq.h"

#define EXPECT(call, st)                                                                   \
    do {                                                                                   \
        const int32_t r_ = (call);                                                         \
        if (r_ != (st)) {                                                                  \
            std::fprintf(stderr, "line %d: %s returned %d, expected %d\n", __LINE__, #call, \
                         (int)r_, (int)(st));                                              \
            return 1;                                                                      \
        }                                                                                  \
    } while (0)

static void *const F = reinterpret_cast<void *>(0x10000);

int main() {
    hatq_conv_desc d = {192, 192, 5, 2, 2, 0, 0, 64};
    int32_t ho = 0, wo = 0;
    EXPECT(hatq_conv_out_hw(&d, 1 << 30, 1 << 30, &ho, &wo), HATQ_OK);
    EXPECT(hatq_conv_out_hw(&d, 1, 1, nullptr, &wo), HATQ_EINVAL);
    hatq_conv_desc big = {1 << 30, 1 << 30, 64, 1, 0, 0, 0, 64};
    (void)hatq_weights_bytes(&big, HATQ_DH);
    hatq_conv_desc bad = {192, 192, 5, 2, 2, 0, 0, 48};
    if (hatq_weights_bytes(&bad, HATQ_DH) != 0) return 1;
    hatq_weights W{};
    W.d = d;
    W.form = HATQ_DH;
    W.cin_pad = 192;
    W.cout_pad = 192;
    W.k_total = 25 * 192;
    W.k_stride = 25 * 192;
    W.pack_stride = 25 * 192;
    W.wq = static_cast<int8_t *>(F);
    W.w_scale = static_cast<float *>(F);
    W.bias = static_cast<float *>(F);
    W.wpack = static_cast<int8_t *>(F);
    const auto *xf = static_cast<const float *>(F);
    auto *xq = static_cast<int8_t *>(F);
    auto *fl = static_cast<float *>(F);
    EXPECT(hatq_prepare_weights(&d, HATQ_DH, xf, nullptr, F, 16, &W, nullptr), HATQ_EWORKSPACE);
    EXPECT(hatq_fwht_quant_act(xf, 1, 4, 4, 48, 32, nullptr, xq, fl, F, 256, nullptr), HATQ_EUNSUPPORTED);
    EXPECT(hatq_fwht_quant_act(xf, 4, 4, 4, 64, 64, nullptr, xq, fl, F, 1, nullptr), HATQ_EWORKSPACE);
    EXPECT(hatq_fwht_quant_act(xf, 1, 1 << 30, 1 << 30, 1 << 30, 3, nullptr, xq, fl, F, 256, nullptr), HATQ_EINVAL);
    EXPECT(hatq_fwht_quant_act_noalloc(xf, HATQ_NOALLOC_MAX_SAMPLES + 1, 4, 4, 64, 64, xq, fl, nullptr),
           HATQ_EUNSUPPORTED);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1, 8, 8, 7, nullptr, F, 0, nullptr, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1, 8, 8, HATQ_OUT_F32, nullptr, F, 0, nullptr, 4, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1, 8, 8, HATQ_OUT_I8, nullptr, F, 64, nullptr, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1, 8, 8, HATQ_OUT_F32, nullptr, F, 128, fl, 0, nullptr), HATQ_EUNSUPPORTED);
    EXPECT(hatq_conv_int8(&W, xq, fl, -1, 8, 8, HATQ_OUT_F32, nullptr, F, 0, nullptr, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1, 0, 8, HATQ_OUT_F32, nullptr, F, 0, nullptr, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1, 8, 8, HATQ_OUT_F32, nullptr, nullptr, 0, nullptr, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8_requant(&W, xq, fl, 1, 8, 8, 3, fl, fl, xq, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_int_transition_params(&W, 0.0f, 1.0f, 64, reinterpret_cast<int32_t *>(F), nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8_int_transition(&W, xq, 1, 8, 8, 64, nullptr, xq, 0, nullptr), HATQ_EINVAL);
    EXPECT(hatq_range_expansion(xf, 65536, 4, 4, 64, 64, fl, nullptr, nullptr, nullptr), HATQ_EINVAL);
    EXPECT(hatq_range_expansion(xf, 1, 1 << 30, 1 << 30, 64, 64, fl, nullptr, nullptr, nullptr), HATQ_EINVAL);
    EXPECT(hatq_fwht_quant_act(xf, 1 << 30, 1 << 30, 1 << 30, 64, 64, nullptr, xq, fl, F, 256, nullptr), HATQ_EINVAL);
    EXPECT(hatq_conv_int8(&W, xq, fl, 1 << 30, 1 << 30, 1 << 30, HATQ_OUT_F32, nullptr, F, 0, nullptr, 0, nullptr),
           HATQ_EINVAL);
    if (hatq_layer_ws_bytes(&W, 1 << 30, 1 << 30, 1 << 30) != 0) return 1;
    int32_t form = -1;
    EXPECT(hatq_select_form(3, 2, 0.8, &form), HATQ_EINVAL);
    EXPECT(hatq_select_form(1, 2, 0.8, &form), HATQ_OK);
    EXPECT(hatq_hadamard_order(0), 0);
    EXPECT(hatq_hadamard_order(4097), 0);
    EXPECT(hatq_hadamard_order(3), 4);
    EXPECT(hatq_hadamard_order(192), 192);
    EXPECT(hatq_hadamard_order(4096), 4096);
    EXPECT(hatq_layer_forward(&W, HATQ_WH, xf, 1, 16, 16, nullptr, fl, nullptr, 0, nullptr, F, 1u << 30, nullptr),
           HATQ_EINVAL);
    EXPECT(hatq_export_weights(&W, nullptr, nullptr, nullptr, nullptr), HATQ_OK);
    hatq_weights Wb = W;
    Wb.k_total += 1;
    EXPECT(hatq_export_weights(&Wb, xq, fl, fl, nullptr), HATQ_EINVAL);
    for (int s = -2; s < 8; ++s)
        if (!hatq_status_string(s)) return 1;
    std::printf("abi driver ok\n");
    return 0;
}
