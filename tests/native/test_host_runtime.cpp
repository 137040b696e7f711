// Native driver of the host runtime under AddressSanitizer / UBSan, linked
// with the stub launchers of host_stub.cpp (no GPU).  Exercises the record
// lifecycle, the ledger, validation failures and injected workspace failure.
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "memsave.h"
#include "memsave_testing.h"

extern "C" const char *stub_violations();

static int g_fail = 0;
#define CHECK(c)                                                              \
    do {                                                                      \
        if (!(c)) {                                                           \
            std::printf("FAIL %s:%d: %s (%s)\n", __FILE__, __LINE__, #c, ms_last_error()); \
            ++g_fail;                                                         \
        }                                                                     \
    } while (0)

static ms_tensor nhwc(int64_t N, int64_t C, int64_t H, int64_t W, void *p) {
    ms_tensor t;
    std::memset(&t, 0, sizeof t);
    t.data = p;
    t.dtype = MS_BF16;
    t.ndim = 4;
    int64_t sh[4] = {N, C, H, W}, st[4] = {H * W * C, 1, W * C, C};
    std::memcpy(t.shape, sh, sizeof sh);
    std::memcpy(t.stride, st, sizeof st);
    return t;
}

static ms_tensor vec1(int64_t n, void *p) {
    ms_tensor t;
    std::memset(&t, 0, sizeof t);
    t.data = p;
    t.dtype = MS_BF16;
    t.ndim = 1;
    t.shape[0] = n;
    t.stride[0] = 1;
    return t;
}

int main() {
    void *P = reinterpret_cast<void *>(uintptr_t(0x7f0000000000ull));
    ms_layer conv;
    std::memset(&conv, 0, sizeof conv);
    conv.kind = MS_CONV2D;
    conv.stride[0] = conv.stride[1] = 1;
    conv.pad[0] = conv.pad[1] = 1;
    ms_tensor x = nhwc(32, 256, 28, 28, P), W = nhwc(256, 256, 3, 3, P), b = vec1(256, P);
    ms_tensor y = nhwc(32, 256, 28, 28, P);

    uint64_t live0, peak0, live, peak;
    CHECK(ms_ledger_read(&live0, &peak0) == MS_OK);
    for (uint32_t mask = 0; mask < 8; ++mask) {
        ms_record *r = nullptr;
        CHECK(ms_layer_forward(&conv, &x, &W, &b, mask, &y, &r, nullptr) == MS_OK);
        if (mask == 0) {
            CHECK(r == nullptr);
            continue;
        }
        ms_account a;
        CHECK(ms_record_account(r, &a) == MS_OK);
        const uint64_t want = (mask & MS_RG_WEIGHT) ? 32ull * 256 * 28 * 28 * 2 : 0;
        CHECK(a.saved_activation_bytes == want);
        CHECK(ms_ledger_read(&live, &peak) == MS_OK);
        CHECK(live - live0 == want);
        ms_tensor gy = nhwc(32, 256, 28, 28, P), gx = nhwc(32, 256, 28, 28, P), gw = nhwc(256, 256, 3, 3, P),
                  gb = vec1(256, P);
        // contradicting grad set
        CHECK(ms_layer_backward(r, &gy, (mask & 1) ? nullptr : &gx, (mask & 2) ? &gw : nullptr,
                                (mask & 4) ? &gb : nullptr, nullptr) == MS_E_MASK);
        if (mask & (MS_RG_WEIGHT | MS_RG_BIAS)) {
            ms_testing_fail_next_workspace(1);
            CHECK(ms_layer_backward(r, &gy, (mask & 1) ? &gx : nullptr, (mask & 2) ? &gw : nullptr,
                                    (mask & 4) ? &gb : nullptr, nullptr) == MS_E_NOMEM);
            CHECK(ms_ledger_read(&live, &peak) == MS_OK);
            CHECK(live - live0 == want);
        }
        CHECK(ms_layer_backward(r, &gy, (mask & 1) ? &gx : nullptr, (mask & 2) ? &gw : nullptr,
                                (mask & 4) ? &gb : nullptr, nullptr) == MS_OK);
        CHECK(ms_layer_backward(r, &gy, (mask & 1) ? &gx : nullptr, (mask & 2) ? &gw : nullptr,
                                (mask & 4) ? &gb : nullptr, nullptr) == MS_E_CONSUMED);
        CHECK(ms_ledger_read(&live, &peak) == MS_OK);
        CHECK(live == live0);
        ms_record_free(r);
    }
    // record freed without backward releases its bytes
    ms_record *r = nullptr;
    CHECK(ms_layer_forward(&conv, &x, &W, &b, MS_RG_WEIGHT, &y, &r, nullptr) == MS_OK);
    ms_record_free(r);
    CHECK(ms_ledger_read(&live, &peak) == MS_OK);
    CHECK(live == live0);
    ms_record_free(nullptr);
    // validation errors
    CHECK(ms_layer_forward(nullptr, &x, &W, &b, 1, &y, &r, nullptr) == MS_E_NULL);
    CHECK(ms_layer_forward(&conv, &x, &W, &b, 9, &y, &r, nullptr) == MS_E_MASK);
    CHECK(ms_layer_forward(&conv, &x, &W, &b, 1, &y, nullptr, nullptr) == MS_E_NULL);
    ms_tensor xbad = x;
    xbad.stride[1] = -1;   // any layout is staged, but strides must not be negative
    CHECK(ms_layer_forward(&conv, &xbad, &W, &b, 1, &y, &r, nullptr) == MS_E_LAYOUT);
    ms_tensor ybad = y;
    ybad.stride[2] = 0;    // an output may not overlap itself
    CHECK(ms_layer_forward(&conv, &x, &W, &b, 1, &ybad, &r, nullptr) == MS_E_LAYOUT);
    CHECK(ms_layer_backward(nullptr, &y, nullptr, nullptr, nullptr, nullptr) == MS_E_NULL);
    ms_account acct;
    CHECK(ms_policy_account(&conv, &x, &W, &b, 1, 7, &acct) == MS_E_ARG);
    CHECK(ms_policy_account(&conv, &x, &W, &b, 1, MS_POLICY_PYTORCH_DEFAULT, &acct) == MS_OK);
    CHECK(acct.saved_activation_bytes == 32ull * 256 * 28 * 28 * 2);
    CHECK(std::strcmp(ms_status_str(MS_E_CONSUMED), "record already consumed") == 0);
    CHECK(ms_testing_live_records() == 0);
    CHECK(std::strlen(stub_violations()) == 0);
    if (g_fail) {
        std::printf("%d failures\n", g_fail);
        return 1;
    }
    std::printf("ALL OK\n");
    return 0;
}
