/* Runs every function of the oracle (oracle/mfpsn_oracle.c, built with
 * AddressSanitizer and UndefinedBehaviorSanitizer) on small inputs that reach
 * its edge cases: empty sequences, orders longer than the sequence, dilations
 * past its end, the extreme shift ranges of the float and Q8.8 paths, the
 * most negative Q8.8 inputs, special float values, per-channel thresholds,
 * step-by-step rings that start as garbage, and the batch-normalized step.
 * Any out-of-bounds access, signed overflow or invalid shift aborts the run.
 * Test infrastructure only.  Prints "oracle driver: OK" and exits 0. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

float orc_exp(float y);
float orc_surrogate(int kind, float alpha, float u);
uint16_t orc_f32_to_bf16(float f);
float orc_bf16_to_f32(uint16_t h);
void orc_quantize(const float* w, int64_t count, int lo, int hi, int8_t* sign, int8_t* shift);
void orc_quantizer_grad(const float* w, const int8_t* shift, int lo, int hi, const float* grad_wq, int64_t count,
                        int mode, float* grad_w);
void orc_forward_f32(const float* x, int T, int N, int C, int S, int k, int d, const int8_t* sign,
                     const int8_t* shift, int lo, int hi, const float* bias, float v_th, const float* v_th_c,
                     float* H, uint8_t* spikes, int64_t* tap_count);
void orc_forward_q88(const int16_t* x, int T, int N, int C, int S, int k, int d, const int8_t* sign,
                     const int8_t* shift, int lo, int hi, const int32_t* bias, int32_t v_th,
                     const int32_t* v_th_c, int32_t* H, uint8_t* spikes, int64_t* tap_count);
void orc_backward_f32(const float* x, const float* grad_spikes, int T, int N, int C, int S, int k, int d,
                      const int8_t* sign, const int8_t* shift, int lo, int hi, const float* bias, float v_th,
                      const float* v_th_c, int kind, float alpha, float* H, float* dH, float* grad_x,
                      double* grad_w, double* grad_b, double* grad_vth);
int32_t orc_surrogate_q15(int kind, float alpha, int32_t u);
void orc_backward_q88(const int16_t* x, const int16_t* grad_spikes, int T, int N, int C, int S, int k, int d,
                      const int8_t* sign, const int8_t* shift, int lo, int hi, const int32_t* bias, int32_t v_th,
                      const int32_t* v_th_c, int kind, float alpha, int32_t* H, int32_t* dH, int32_t* grad_x,
                      int64_t* grad_w, int64_t* grad_b, int64_t* grad_vth);
void orc_stream_step_f32(const float* x_t, int N, int C, int S, int k, int d, int64_t t, float* hist,
                         const int8_t* sign, const int8_t* shift, int lo, int hi, const float* bias, float v_th,
                         float* H_t, uint8_t* spikes_t);
void orc_stream_step_q88(const int16_t* x_t, int N, int C, int S, int k, int d, int64_t t, int16_t* hist,
                         const int8_t* sign, const int8_t* shift, int lo, int hi, const int32_t* bias,
                         int32_t v_th, int32_t* H_t, uint8_t* spikes_t);
void orc_bn_forward_stats(const float* x, int T, int N, int C, int S, int k, int d, const float* w,
                          const float* gamma, const float* beta, float eps, float* w_f, float* b_f, double* aux,
                          double* stats);
void orc_bn_backward(const float* x, int T, int N, int C, int S, int k, int d, const float* w, const float* gamma,
                     float eps, const double* aux, const double* grad_wf, const double* grad_bf,
                     const double* grad_xq, double* grad_x, double* grad_w, double* grad_gamma,
                     double* grad_beta);
int orc_sawtooth_dilation(int layer, int period);

static uint32_t rng = 12345u;
static uint32_t next(void)
{
    rng = rng * 1664525u + 1013904223u;
    return rng;
}
static float unit(void) { return (float)(next() >> 8) / 16777216.0f * 2.0f - 1.0f; }

/* exact-size heap buffers, so AddressSanitizer sees every overrun */
#define ALLOC(type, n) ((type*)malloc(sizeof(type) * (size_t)((n) > 0 ? (n) : 1)))

static void run_float(int T, int N, int C, int S, int k, int d, int lo, int hi, int specials)
{
    const int64_t n = (int64_t)T * N * C * S;
    float *x = ALLOC(float, n), *g = ALLOC(float, n), *H = ALLOC(float, n), *dH = ALLOC(float, n);
    float *gx = ALLOC(float, n), *bias = ALLOC(float, C), *vc = ALLOC(float, C);
    uint8_t* spk = ALLOC(uint8_t, n);
    int8_t *sign = ALLOC(int8_t, C * k), *shift = ALLOC(int8_t, C * k);
    double *gw = ALLOC(double, C * k), *gb = ALLOC(double, C), *gv = ALLOC(double, C);
    const float sp[] = {0.0f, -0.0f, 1e-45f, -1e-40f, 3e38f, -3e38f, INFINITY, -INFINITY, NAN, 1e-30f};
    for (int64_t i = 0; i < n; ++i) {
        x[i] = unit() * 4.0f;
        g[i] = unit();
        if (specials && next() % 7 == 0)
            x[i] = sp[next() % 10];
        if (specials && next() % 11 == 0)
            g[i] = sp[next() % 10];
    }
    for (int i = 0; i < C * k; ++i) {
        sign[i] = (next() & 1) ? 1 : -1;
        shift[i] = (int8_t)(lo + (int)(next() % (uint32_t)(hi - lo + 1)));
    }
    for (int c = 0; c < C; ++c) {
        bias[c] = unit();
        vc[c] = unit();
    }
    int64_t taps = 0;
    for (int per = 0; per < 2; ++per) {
        orc_forward_f32(x, T, N, C, S, k, d, sign, shift, lo, hi, bias, 0.5f, per ? vc : NULL, H, spk, &taps);
        for (int kind = 0; kind < 3; ++kind)
            orc_backward_f32(x, g, T, N, C, S, k, d, sign, shift, lo, hi, bias, 0.5f, per ? vc : NULL, kind, 4.0f,
                             H, dH, gx, gw, gb, per ? gv : NULL);
    }
    /* step by step from a garbage ring */
    if (N * C * S > 0) {
        const int64_t M = (int64_t)N * C * S, R = (int64_t)(k - 1) * d + 1;
        float* hist = ALLOC(float, R * M);
        for (int64_t i = 0; i < R * M; ++i)
            hist[i] = NAN;
        for (int t = 0; t < T; ++t)
            orc_stream_step_f32(x + t * M, N, C, S, k, d, t, hist, sign, shift, lo, hi, bias, 0.5f, H, spk);
        free(hist);
    }
    free(x); free(g); free(H); free(dH); free(gx); free(bias); free(vc); free(spk); free(sign); free(shift);
    free(gw); free(gb); free(gv);
}

static void run_q88(int T, int N, int C, int S, int k, int d, int lo, int hi)
{
    const int64_t n = (int64_t)T * N * C * S;
    int16_t *x = ALLOC(int16_t, n), *g = ALLOC(int16_t, n);
    int32_t *H = ALLOC(int32_t, n), *dH = ALLOC(int32_t, n), *gx = ALLOC(int32_t, n);
    int32_t *bias = ALLOC(int32_t, C), *vc = ALLOC(int32_t, C);
    uint8_t* spk = ALLOC(uint8_t, n);
    int8_t *sign = ALLOC(int8_t, C * k), *shift = ALLOC(int8_t, C * k);
    int64_t *gw = ALLOC(int64_t, C * k), *gb = ALLOC(int64_t, C), *gv = ALLOC(int64_t, C);
    for (int64_t i = 0; i < n; ++i) {
        x[i] = (int16_t)(next() % 3 == 0 ? -32768 : (int)(next() & 0xFFFF) - 32768);
        g[i] = (int16_t)(next() % 3 == 0 ? -32768 : (int)(next() & 0xFFFF) - 32768);
    }
    for (int i = 0; i < C * k; ++i) {
        sign[i] = (next() & 1) ? 1 : -1;
        shift[i] = (int8_t)(lo + (int)(next() % (uint32_t)(hi - lo + 1)));
    }
    for (int c = 0; c < C; ++c) {
        bias[c] = (int32_t)(next() % 2001) - 1000;
        vc[c] = (int32_t)(next() % 4001) - 2000;
    }
    for (int per = 0; per < 2; ++per) {
        orc_forward_q88(x, T, N, C, S, k, d, sign, shift, lo, hi, bias, 256, per ? vc : NULL, H, spk, NULL);
        for (int kind = 0; kind < 3; ++kind)
            orc_backward_q88(x, g, T, N, C, S, k, d, sign, shift, lo, hi, bias, 256, per ? vc : NULL, kind, 4.0f, H,
                             dH, gx, gw, gb, per ? gv : NULL);
    }
    if (N * C * S > 0) {
        const int64_t M = (int64_t)N * C * S, R = (int64_t)(k - 1) * d + 1;
        int16_t* hist = ALLOC(int16_t, R * M);
        for (int64_t i = 0; i < R * M; ++i)
            hist[i] = 0x5A5A;
        for (int t = 0; t < T; ++t)
            orc_stream_step_q88(x + t * M, N, C, S, k, d, t, hist, sign, shift, lo, hi, bias, 256, H, spk);
        free(hist);
    }
    free(x); free(g); free(H); free(dH); free(gx); free(bias); free(vc); free(spk); free(sign); free(shift);
    free(gw); free(gb); free(gv);
}

static void run_bn(int T, int N, int C, int S, int k, int d)
{
    const int64_t n = (int64_t)T * N * C * S;
    float *x = ALLOC(float, n), *w = ALLOC(float, C * k), *gamma = ALLOC(float, C), *beta = ALLOC(float, C);
    float *w_f = ALLOC(float, C * k), *b_f = ALLOC(float, C);
    double *aux = ALLOC(double, 4 * C), *stats = ALLOC(double, 2 * C), *gwf = ALLOC(double, C * k);
    double *gbf = ALLOC(double, C), *gxq = ALLOC(double, n), *gx = ALLOC(double, n), *gw = ALLOC(double, C * k);
    double *gg = ALLOC(double, C), *gbeta = ALLOC(double, C);
    for (int64_t i = 0; i < n; ++i) {
        x[i] = unit() * 1000.0f + 3000.0f;  /* a large mean against the spread */
        gxq[i] = unit();
    }
    for (int i = 0; i < C * k; ++i) {
        w[i] = unit();
        gwf[i] = unit();
    }
    for (int c = 0; c < C; ++c) {
        gamma[c] = 1.0f;
        beta[c] = -1.0f;
        gbf[c] = unit();
    }
    orc_bn_forward_stats(x, T, N, C, S, k, d, w, gamma, beta, 1e-5f, w_f, b_f, aux, stats);
    orc_bn_backward(x, T, N, C, S, k, d, w, gamma, 1e-5f, aux, gwf, gbf, gxq, gx, gw, gg, gbeta);
    free(x); free(w); free(gamma); free(beta); free(w_f); free(b_f); free(aux); free(stats); free(gwf);
    free(gbf); free(gxq); free(gx); free(gw); free(gg); free(gbeta);
}

int main(void)
{
    /* elementary functions over their whole domains */
    for (int i = -2000; i <= 2000; ++i) {
        volatile float y = orc_exp((float)i * 0.05f);
        volatile float s = orc_surrogate(i % 3 < 0 ? -(i % 3) : i % 3, 4.0f, (float)i * 0.01f);
        volatile int32_t q = orc_surrogate_q15(0, 4.0f, i * 1000);
        (void)y; (void)s; (void)q;
    }
    (void)orc_exp(NAN);
    (void)orc_exp(INFINITY);
    (void)orc_exp(-INFINITY);
    (void)orc_surrogate_q15(1, 1024.0f, INT32_MAX);
    (void)orc_surrogate_q15(2, 0.0f, INT32_MIN + 1);
    for (uint32_t b = 0; b < 0x10000u; b += 7)
        (void)orc_f32_to_bf16(orc_bf16_to_f32((uint16_t)b));
    /* quantizer and its gradient on special values and the extreme ranges */
    {
        const float w[] = {0.0f, -0.0f, INFINITY, -INFINITY, NAN, 1e-45f, -1e-38f, 3e38f, 1.41421354f, -0.7f, 1.0f};
        const int cnt = (int)(sizeof(w) / sizeof(w[0]));
        int8_t sign[16], shift[16];
        float gq[16], gw[16];
        for (int i = 0; i < cnt; ++i)
            gq[i] = 1.0f;
        const int ranges[][2] = {{-128, 127}, {0, 7}, {-126, 126}, {127, 127}, {-128, -128}};
        for (int r = 0; r < 5; ++r) {
            orc_quantize(w, cnt, ranges[r][0], ranges[r][1], sign, shift);
            orc_quantizer_grad(w, shift, ranges[r][0], ranges[r][1], gq, cnt, 1, gw);
            orc_quantizer_grad(w, shift, ranges[r][0], ranges[r][1], gq, cnt, 0, gw);
        }
    }
    for (int l = 0; l < 50; ++l)
        (void)orc_sawtooth_dilation(l, 1 + l % 5);
    /* the training step: empty, short, long-receptive-field and ragged shapes */
    run_float(0, 2, 3, 1, 4, 2, 0, 7, 0);
    run_float(5, 0, 3, 2, 4, 2, 0, 7, 0);
    run_float(1, 2, 3, 2, 8, 3, 0, 7, 1);
    run_float(9, 2, 3, 2, 5, 7, -126, 126, 1);
    run_float(13, 3, 2, 5, 32, 1, 0, 7, 1);
    run_float(17, 2, 4, 3, 3, 2, -20, 120, 1);
    run_float(11, 1, 2, 1, 1, 1, 126, 126, 1);
    run_q88(0, 2, 3, 1, 4, 2, 0, 7);
    run_q88(7, 2, 3, 2, 6, 3, 0, 31);
    run_q88(15, 3, 2, 2, 32, 1, 0, 0);
    run_q88(9, 2, 2, 3, 4, 9, 31, 31);
    run_bn(13, 2, 3, 2, 4, 2);
    run_bn(6, 3, 2, 1, 8, 3);
    run_bn(0, 2, 2, 1, 3, 1);
    printf("oracle driver: OK\n");
    return 0;
}
