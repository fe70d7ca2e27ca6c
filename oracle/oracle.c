/*
 * CPU oracle for sliced DNN inference (MOPAR, arXiv 2404.02445).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow reference that the
 * GPU library is checked against.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it; the product path never does.
 * It shares no code, header or table with the GPU library.
 *
 * Every routine is the textbook definition of the layer it names, written
 * as direct loops: accumulation in double, then one rounding of each stored
 * result to the storage type (rnd = 0: keep double, 1: binary32,
 * 2: bfloat16, both round-to-nearest-even).  Layouts are PyTorch's: images
 * [N][C][H][W], sequences [B][S][F], linear weights [out][in], conv weights
 * [C_out][C_in][kh][kw], LSTM weights [4H][in] in gate order i, f, g, o.
 *
 * The layers are those of the models the paper evaluates (Sec. II-A names
 * VGG, ResNet, LSTM and BERT; Sec. IV lists the services); the paper defines
 * none of them itself, so each follows its standard definition:
 *   conv2d, max-pool, global average pool, linear  (VGG, ResNet)
 *   layer norm, multi-head self-attention, GELU     (BERT, post-LN)
 *   LSTM cell                                        (PyTorch gate convention)
 * The boundary codec is the one-layer-encoder / one-layer-decoder
 * autoencoder of Sec. III-D (COM), read as a 1x1 convolution over channels
 * at every position: code = W_e x + b_e, y = W_d code + b_d.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <stdlib.h>

#define OR_API __attribute__((visibility("default")))

enum { ACT_NONE = 0, ACT_RELU = 1, ACT_GELU = 2 };

/* ---- storage rounding ------------------------------------------------- */

/* Round to the nearest bfloat16 value (8 significant bits, binary32
 * exponent range, subnormal quantum 2^-133), ties to even. */
static double round_bf16(double x) {
    if (x == 0.0 || !isfinite(x)) return x;
    int e;
    frexp(x, &e);                 /* x = f * 2^e with 0.5 <= |f| < 1 */
    int q = e - 8;                /* weight of the last kept bit */
    if (q < -133) q = -133;
    double r = ldexp(nearbyint(ldexp(x, -q)), q);   /* default mode: ties to even */
    if (fabs(r) > 3.3895313892515355e38) r = copysign(INFINITY, x);
    return r;
}

OR_API double or_round1(double x, int rnd) {
    if (rnd == 1) return (double)(float)x;   /* C conversion rounds to nearest even */
    if (rnd == 2) return round_bf16(x);
    return x;
}

OR_API void or_round(double* x, int64_t n, int rnd) {
    for (int64_t i = 0; i < n; ++i) x[i] = or_round1(x[i], rnd);
}

static double activate(double v, int act) {
    if (act == ACT_RELU) return v > 0.0 ? v : 0.0;
    if (act == ACT_GELU) return 0.5 * v * (1.0 + erf(v / sqrt(2.0)));
    return v;
}

/* ---- conv2d ------------------------------------------------------------
 * y[n,co,ho,wo] = act( b[co] + sum_{ci,r,s} w[co,ci,r,s] * x[n,ci,ho*st-p+r,wo*st-p+s]
 *                      + res[n,co,ho,wo] ), zero padding outside the image. */
OR_API void or_conv2d(const double* x, int64_t N, int64_t C, int64_t H, int64_t W,
                      const double* w, const double* b, int64_t Co, int64_t kh, int64_t kw,
                      int64_t st, int64_t pad, const double* res, int act, int rnd, double* y) {
    const int64_t Ho = (H + 2 * pad - kh) / st + 1, Wo = (W + 2 * pad - kw) / st + 1;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t co = 0; co < Co; ++co) {
            double* acc = (double*)malloc(sizeof(double) * Ho * Wo);
            for (int64_t i = 0; i < Ho * Wo; ++i) acc[i] = b ? b[co] : 0.0;
            for (int64_t ci = 0; ci < C; ++ci)
                for (int64_t r = 0; r < kh; ++r)
                    for (int64_t s = 0; s < kw; ++s) {
                        const double wv = w[((co * C + ci) * kh + r) * kw + s];
                        const double* xp = x + (n * C + ci) * H * W;
                        for (int64_t ho = 0; ho < Ho; ++ho) {
                            const int64_t hi = ho * st - pad + r;
                            if (hi < 0 || hi >= H) continue;
                            for (int64_t wo = 0; wo < Wo; ++wo) {
                                const int64_t wi = wo * st - pad + s;
                                if (wi < 0 || wi >= W) continue;
                                acc[ho * Wo + wo] += wv * xp[hi * W + wi];
                            }
                        }
                    }
            double* yp = y + (n * Co + co) * Ho * Wo;
            const double* rp = res ? res + (n * Co + co) * Ho * Wo : NULL;
            for (int64_t i = 0; i < Ho * Wo; ++i)
                yp[i] = or_round1(activate(acc[i] + (rp ? rp[i] : 0.0), act), rnd);
            free(acc);
        }
}

/* ---- pooling ------------------------------------------------------------ */

/* Max over the k x k window; positions outside the image count as -inf. */
OR_API void or_maxpool2d(const double* x, int64_t N, int64_t C, int64_t H, int64_t W,
                         int64_t k, int64_t st, int64_t pad, double* y) {
    const int64_t Ho = (H + 2 * pad - k) / st + 1, Wo = (W + 2 * pad - k) / st + 1;
    #pragma omp parallel for collapse(2)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c)
            for (int64_t ho = 0; ho < Ho; ++ho)
                for (int64_t wo = 0; wo < Wo; ++wo) {
                    double m = -INFINITY;
                    for (int64_t r = 0; r < k; ++r)
                        for (int64_t s = 0; s < k; ++s) {
                            const int64_t hi = ho * st - pad + r, wi = wo * st - pad + s;
                            if (hi < 0 || hi >= H || wi < 0 || wi >= W) continue;
                            const double v = x[((n * C + c) * H + hi) * W + wi];
                            if (v > m) m = v;
                        }
                    y[((n * C + c) * Ho + ho) * Wo + wo] = m;
                }
}

/* Global average: y[n,c] = (sum over H*W) / (H*W). */
OR_API void or_avgpool_global(const double* x, int64_t N, int64_t C, int64_t H, int64_t W,
                              int rnd, double* y) {
    for (int64_t n = 0; n < N; ++n)
        for (int64_t c = 0; c < C; ++c) {
            double s = 0.0;
            for (int64_t i = 0; i < H * W; ++i) s += x[(n * C + c) * H * W + i];
            y[n * C + c] = or_round1(s / (double)(H * W), rnd);
        }
}

/* ---- linear ---------------------------------------------------------------
 * y[m,n] = act( b[n] + sum_k x[m,k] * w[n,k] + res[m,n] ). */
OR_API void or_linear(const double* x, int64_t M, int64_t K, const double* w, const double* b,
                      int64_t Nout, const double* res, int act, int rnd, double* y) {
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < Nout; ++n) {
            double acc = b ? b[n] : 0.0;
            const double* xr = x + m * K;
            const double* wr = w + n * K;
            for (int64_t k = 0; k < K; ++k) acc += xr[k] * wr[k];
            if (res) acc += res[m * Nout + n];
            y[m * Nout + n] = or_round1(activate(acc, act), rnd);
        }
}

/* ---- layer norm -----------------------------------------------------------
 * v = x (+ res); y = (v - mean) / sqrt(var + eps) * g + beta, var biased. */
OR_API void or_layernorm(const double* x, const double* res, int64_t M, int64_t F,
                         const double* g, const double* beta, double eps, int rnd, double* y) {
    #pragma omp parallel for
    for (int64_t m = 0; m < M; ++m) {
        double* v = (double*)malloc(sizeof(double) * F);
        double mean = 0.0, var = 0.0;
        for (int64_t f = 0; f < F; ++f) { v[f] = x[m * F + f] + (res ? res[m * F + f] : 0.0); mean += v[f]; }
        mean /= (double)F;
        for (int64_t f = 0; f < F; ++f) var += (v[f] - mean) * (v[f] - mean);
        var /= (double)F;
        const double inv = 1.0 / sqrt(var + eps);
        for (int64_t f = 0; f < F; ++f) y[m * F + f] = or_round1((v[f] - mean) * inv * g[f] + beta[f], rnd);
        free(v);
    }
}

/* ---- multi-head self-attention -----------------------------------------
 * qkv[b,s,:] = [Q | K | V], each F = heads*d wide, head h at columns h*d..h*d+d-1.
 * For each (b, h, i): p = softmax_j(scale * <q_i, k_j>) (max subtracted),
 * y[b,i,h*d+e] = sum_j p_j v[j,e].  No mask. */
OR_API void or_attention(const double* qkv, int64_t B, int64_t S, int64_t heads, int64_t d,
                         double scale, int rnd, double* y) {
    const int64_t F = heads * d;
    #pragma omp parallel for collapse(3)
    for (int64_t b = 0; b < B; ++b)
        for (int64_t h = 0; h < heads; ++h)
            for (int64_t i = 0; i < S; ++i) {
                double* p = (double*)malloc(sizeof(double) * S);
                const double* q = qkv + (b * S + i) * 3 * F + h * d;
                double mx = -INFINITY;
                for (int64_t j = 0; j < S; ++j) {
                    const double* kk = qkv + (b * S + j) * 3 * F + F + h * d;
                    double s = 0.0;
                    for (int64_t e = 0; e < d; ++e) s += q[e] * kk[e];
                    p[j] = s * scale;
                    if (p[j] > mx) mx = p[j];
                }
                double den = 0.0;
                for (int64_t j = 0; j < S; ++j) { p[j] = exp(p[j] - mx); den += p[j]; }
                for (int64_t e = 0; e < d; ++e) {
                    double o = 0.0;
                    for (int64_t j = 0; j < S; ++j) o += p[j] * qkv[(b * S + j) * 3 * F + 2 * F + h * d + e];
                    y[(b * S + i) * F + h * d + e] = or_round1(o / den, rnd);
                }
                free(p);
            }
}

/* ---- embeddings -----------------------------------------------------------
 * BERT: v = tok[id] + pos[s] + type[0], then layer norm. */
OR_API void or_embed_bert(const int32_t* ids, int64_t B, int64_t S, const double* tok,
                          const double* pos, const double* type, int64_t F, const double* g,
                          const double* beta, double eps, int rnd, double* y) {
    double* v = (double*)malloc(sizeof(double) * B * S * F);
    for (int64_t b = 0; b < B; ++b)
        for (int64_t s = 0; s < S; ++s)
            for (int64_t f = 0; f < F; ++f)
                v[(b * S + s) * F + f] = tok[(int64_t)ids[b * S + s] * F + f] + pos[s * F + f] + type[f];
    or_layernorm(v, NULL, B * S, F, g, beta, eps, rnd, y);
    free(v);
}

/* Plain gather: y[i,:] = table[id_i,:]. */
OR_API void or_embed(const int32_t* ids, int64_t n, const double* table, int64_t F, double* y) {
    for (int64_t i = 0; i < n; ++i) memcpy(y + i * F, table + (int64_t)ids[i] * F, sizeof(double) * F);
}

/* ---- LSTM (one layer, h_0 = c_0 = 0) --------------------------------------
 * g = W_ih x_t + b_ih + W_hh h_{t-1} + b_hh, split [i | f | g | o];
 * c_t = sig(f) c_{t-1} + sig(i) tanh(g);  h_t = sig(o) tanh(c_t).
 * Stored: h_t rounded to the storage type (rnd), c_t to binary32 (when rnd != 0). */
static double sigm(double v) { return 1.0 / (1.0 + exp(-v)); }

OR_API void or_lstm(const double* x, int64_t B, int64_t T, int64_t E, int64_t Hd,
                    const double* w_ih, const double* w_hh, const double* b_ih, const double* b_hh,
                    int rnd, double* y) {
    double* h = (double*)malloc(sizeof(double) * Hd);
    double* c = (double*)malloc(sizeof(double) * Hd);
    double* g = (double*)malloc(sizeof(double) * 4 * Hd);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t u = 0; u < Hd; ++u) h[u] = c[u] = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double* xt = x + (b * T + t) * E;
            #pragma omp parallel for schedule(static)
            for (int64_t r = 0; r < 4 * Hd; ++r) {
                double a = b_ih[r] + b_hh[r];
                for (int64_t e = 0; e < E; ++e) a += w_ih[r * E + e] * xt[e];
                for (int64_t k = 0; k < Hd; ++k) a += w_hh[r * Hd + k] * h[k];
                g[r] = a;
            }
            for (int64_t u = 0; u < Hd; ++u) {
                const double ig = sigm(g[u]), fg = sigm(g[Hd + u]);
                const double gg = tanh(g[2 * Hd + u]);
                c[u] = or_round1(fg * c[u] + ig * gg, rnd ? 1 : 0);
            }
            for (int64_t u = 0; u < Hd; ++u) {
                h[u] = or_round1(sigm(g[3 * Hd + u]) * tanh(c[u]), rnd);
                y[(b * T + t) * Hd + u] = h[u];
            }
        }
    }
    free(h); free(c); free(g);
}

/* ---- autoencoder boundary codec (Sec. III-D) --------------------------------
 * Tensor viewed as x[n][c][l] (images: l = h*W + w; sequences: N = B*S, L = 1).
 * encode: code[n][e][l] = b_e[e] + sum_c W_e[e][c] x[n][c][l]
 * decode: y[n][c][l]    = b_d[c] + sum_e W_d[c][e] code[n][e][l]              */
OR_API void or_ae_apply(const double* x, int64_t N, int64_t Cin, int64_t L, const double* w,
                        const double* b, int64_t Cout, int rnd, double* y) {
    #pragma omp parallel for collapse(2)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t o = 0; o < Cout; ++o)
            for (int64_t l = 0; l < L; ++l) {
                double acc = b[o];
                for (int64_t c = 0; c < Cin; ++c) acc += w[o * Cin + c] * x[(n * Cin + c) * L + l];
                y[(n * Cout + o) * L + l] = or_round1(acc, rnd);
            }
}
