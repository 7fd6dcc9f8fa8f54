// Drives every C-ABI entry point of libmfpsn.so's host layer (built with
// AddressSanitizer and UndefinedBehaviorSanitizer, the GPU launchers replaced
// by counting stubs): invalid arguments must return the documented status
// and launch nothing; valid ones, including sizes at the limits of the
// 32-bit fields, must validate without overflow or out-of-bounds access.
// Test infrastructure only (C, so that device pointers pass as void*).  Prints "abi driver: OK" and exits 0 on success.
#include <stdint.h>
#include <stdio.h>
#include <math.h>
#include <stdlib.h>

#include "mfpsn.h"

extern long stub_launches;

static int failures = 0;
#define EXPECT(call, want)                                                                      \
    do {                                                                                        \
        const long before = stub_launches;                                                      \
        const int got = (call);                                                                 \
        if (got != (want)) {                                                                    \
            fprintf(stderr, "line %d: %s returned %d, expected %d\n", __LINE__, #call, got, want); \
            ++failures;                                                                         \
        }                                                                                       \
        if ((want) != MFPSN_OK && stub_launches != before) {                                    \
            fprintf(stderr, "line %d: %s launched work although it failed\n", __LINE__, #call);  \
            ++failures;                                                                         \
        }                                                                                       \
    } while (0)

static mfpsn_desc desc(int T, int N, int C, int S, int k, int d, int dtype)
{
    mfpsn_desc x;
    x.T = T;
    x.N = N;
    x.C = C;
    x.S = S;
    x.k = k;
    x.dilation = d;
    x.dtype = dtype;
    x.surrogate = MFPSN_SG_SIGMOID;
    x.alpha = 4.0f;
    x.v_th = 1.0f;
    x.v_th_q = 256;
    x.shift_lo = 0;
    x.shift_hi = 7;
    return x;
}

int main()
{
    // fake device addresses: never dereferenced by the host layer
    void* const P = (void*)(uintptr_t)0x10000000;
    char* const Pc = (char*)P;
    const int32_t BIG = 2147483647;
    if (mfpsn_abi_version() != MFPSN_ABI_VERSION)
        ++failures;
    for (int s = -10; s <= 2; ++s)
        if (mfpsn_status_string(s) == NULL)
            ++failures;
    if (mfpsn_sawtooth_dilation(5, 3) != 3 || mfpsn_sawtooth_dilation(-1, 3) != 0 ||
        mfpsn_sawtooth_dilation(BIG, BIG) != 1 || mfpsn_sawtooth_dilation(BIG - 1, BIG) != BIG ||
        mfpsn_sawtooth_dilation(3, 0) != 0)
        ++failures;

    // descriptors at and beyond the limits of every field
    const mfpsn_desc ok = desc(16, 2, 64, 1, 4, 2, MFPSN_F32);
    const int dt[3] = {MFPSN_F32, MFPSN_BF16, MFPSN_Q8_8};
    for (int i = 0; i < 3; ++i) {
        mfpsn_desc d = desc(BIG, 1, 1, 1, 32, BIG, dt[i]);
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_PARAM);
        d = desc(BIG, BIG, BIG, BIG, 32, 1, dt[i]);
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_SHAPE);
        d = desc(BIG, 1, 64, 1, 32, 1 << 20, dt[i]);
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_SHAPE);
        d = desc(BIG, 1, 64, 1, 2, 1, dt[i]);
        size_t n = 0;
        EXPECT(mfpsn_backward_workspace_size(&d, &n), MFPSN_OK);
        d = desc(16, 1 << 14, 1 << 14, 1, 8, 1, dt[i]);
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_SHAPE);
        d = ok;
        d.dtype = dt[i];
        d.k = 0;
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_PARAM);
        d.k = 33;
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_PARAM);
        d.k = 4;
        d.shift_lo = -200;
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_PARAM);
        d.shift_lo = 0;
        d.v_th_q = INT32_MIN;
        d.v_th = INFINITY;
        EXPECT(mfpsn_forward(&d, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_PARAM);
    }
    // valid calls reach the launchers; empty ones launch nothing
    {
        mfpsn_desc d = ok;
        EXPECT(mfpsn_forward(&d, P, P, P, P, P, P, P, P, NULL), MFPSN_OK);
        size_t need = 0;
        EXPECT(mfpsn_backward_workspace_size(&d, &need), MFPSN_OK);
        EXPECT(mfpsn_backward(&d, P, P, NULL, NULL, P, P, P, P, P, P, P, P, P, need, NULL), MFPSN_OK);
        EXPECT(mfpsn_backward(&d, P, P, NULL, NULL, P, P, P, P, P, P, P, P, P, need - 8, NULL),
               MFPSN_ERR_WORKSPACE);
        EXPECT(mfpsn_backward(&d, P, P, NULL, NULL, P, P, P, (void*)(Pc + 2), P, P, P, P, P, need, NULL),
               MFPSN_ERR_ALIGN);
        EXPECT(mfpsn_backward(&d, P, P, NULL, NULL, P, P, P, NULL, P, NULL, P, NULL, P, need, NULL),
               MFPSN_ERR_NULL);
        d.T = 0;
        const long before = stub_launches;
        EXPECT(mfpsn_forward(&d, NULL, P, P, P, NULL, NULL, NULL, NULL, NULL), MFPSN_OK);
        if (stub_launches != before)
            ++failures;
        mfpsn_desc q = desc(1 << 16, 1 << 16, 1, 1, 4, 1, MFPSN_Q8_8);
        EXPECT(mfpsn_backward(&q, P, P, NULL, NULL, P, P, P, NULL, P, P, P, NULL, P, (size_t)1 << 40,
                              NULL),
               MFPSN_ERR_SHAPE);
        q.v_th_q = (1 << 30) + 1;
        EXPECT(mfpsn_forward(&q, P, P, P, P, NULL, P, NULL, NULL, NULL), MFPSN_ERR_PARAM);
    }
    // quantizer and its gradient
    EXPECT(mfpsn_quantize_weights(P, -1, 0, 7, P, P, NULL), MFPSN_ERR_SHAPE);
    EXPECT(mfpsn_quantize_weights(P, (int64_t)1 << 40, 0, 7, P, P, NULL),
           MFPSN_ERR_SHAPE);
    EXPECT(mfpsn_quantize_weights(P, 10, 8, 7, P, P, NULL), MFPSN_ERR_PARAM);
    EXPECT(mfpsn_quantize_weights(P, 10, INT32_MIN, INT32_MAX, P, P, NULL),
           MFPSN_ERR_PARAM);
    EXPECT(mfpsn_quantize_weights(P, 10, 0, 7, P, P, NULL), MFPSN_OK);
    EXPECT(mfpsn_quantizer_grad(P, P, 0, 7, P, -3, 1, P, NULL),
           MFPSN_ERR_SHAPE);
    EXPECT(mfpsn_quantizer_grad(P, P, 0, 7, P, 3, 9, P, NULL),
           MFPSN_ERR_PARAM);
    EXPECT(mfpsn_quantizer_grad(P, P, 0, 7, P, 3, 1, P, NULL),
           MFPSN_OK);
    // streaming step
    {
        mfpsn_desc d = ok;
        int32_t steps = 0;
        size_t bytes = 0;
        EXPECT(mfpsn_stream_ring_bytes(&d, &steps, &bytes), MFPSN_OK);
        if (steps != 7 || bytes != (size_t)7 * 2 * 64 * 4)
            ++failures;
        EXPECT(mfpsn_stream_ring_bytes(&d, NULL, NULL), MFPSN_ERR_NULL);
        EXPECT(mfpsn_stream_step(&d, -1, P, P, P, P, P, P, NULL, NULL),
               MFPSN_ERR_PARAM);
        EXPECT(mfpsn_stream_step(&d, INT64_MAX, P, P, P, P, P, P, NULL,
                                 NULL),
               MFPSN_OK);
        d.k = 32;
        d.dilation = BIG;
        EXPECT(mfpsn_stream_ring_bytes(&d, &steps, &bytes), MFPSN_ERR_PARAM);
    }
    // batch-normalized threshold
    {
        mfpsn_desc d = ok;
        size_t n = 0;
        EXPECT(mfpsn_bn_workspace_size(&d, &n), MFPSN_OK);
        EXPECT(mfpsn_bn_forward_stats(&d, P, P, P, P, 1e-5f,
                                      P, P, P, NULL, P, n, NULL),
               MFPSN_OK);
        EXPECT(mfpsn_bn_forward_stats(&d, P, P, P, P, -1.0f,
                                      P, P, P, NULL, P, n, NULL),
               MFPSN_ERR_PARAM);
        EXPECT(mfpsn_bn_backward(&d, P, P, P, 1e-5f, P,
                                 P, P, P, P, P, P, n - 8, NULL),
               MFPSN_ERR_WORKSPACE);
        mfpsn_desc b = d;
        b.dtype = MFPSN_BF16;
        EXPECT(mfpsn_bn_workspace_size(&b, &n), MFPSN_ERR_DTYPE);
        mfpsn_desc big = desc(BIG, 1, 64, 1, 32, 1, MFPSN_F32);
        EXPECT(mfpsn_bn_workspace_size(&big, &n), MFPSN_OK);
    }
    // time-last layout
    {
        mfpsn_desc d = ok;
        size_t n = 0;
        EXPECT(mfpsn_forward_time_last(&d, P, P, P, P, P, NULL, NULL),
               MFPSN_OK);
        EXPECT(mfpsn_backward_time_last_workspace_size(&d, &n), MFPSN_OK);
        EXPECT(mfpsn_backward_time_last(&d, P, P, P, P, P, P, P, P, P, n, NULL),
               MFPSN_OK);
        EXPECT(mfpsn_backward_time_last(&d, P, P, P, P, P, P, P, P, P, n - 8, NULL),
               MFPSN_ERR_WORKSPACE);
        mfpsn_desc big = desc(BIG, 1, 64, 1, 32, 1 << 10, MFPSN_Q8_8);
        EXPECT(mfpsn_backward_time_last(&big, P, P, P, P, P, P, P, P, P, n, NULL),
               MFPSN_ERR_SHAPE);
        EXPECT(mfpsn_forward_time_last(&big, P, P, P, P, P, NULL, NULL),
               MFPSN_OK);
    }
    // chaining
    EXPECT(mfpsn_spikes_to_input(P, -1, MFPSN_F32, P, NULL), MFPSN_ERR_SHAPE);
    EXPECT(mfpsn_spikes_to_input(P, 5, 9, P, NULL), MFPSN_ERR_DTYPE);
    EXPECT(mfpsn_spikes_to_input(P, 5, MFPSN_F32, (void*)(Pc + 2), NULL), MFPSN_ERR_ALIGN);
    EXPECT(mfpsn_spikes_to_input(P, INT64_MAX, MFPSN_Q8_8, P, NULL), MFPSN_OK);
    if (failures) {
        fprintf(stderr, "abi driver: %d failures\n", failures);
        return 1;
    }
    printf("abi driver: OK (%ld launches reached the stubs)\n", stub_launches);
    return 0;
}
