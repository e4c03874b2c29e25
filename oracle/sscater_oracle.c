/*
 * CPU oracle for the delta-scatter backbone -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code, header or table with the GPU
 * library; it is the plain definition that the GPU path must reproduce.
 *
 * SSCATeR (arXiv 2512.08557) claims that its recycled convolution maps are
 * identical to recomputing the sparse / dense convolution from scratch
 * (abstract; Sec. IV-G "Performance and Results Evaluation"; Sec. V).  So the
 * oracle does not model the method at all: for one window it recomputes every
 * backbone layer densely, in double precision, from the input canvas.
 *
 *   Z_l[y,x,co] = sum_{m,n in 0..2} sum_ci Y_{l-1}[s*y+m-1, s*x+n-1, ci] * W_l[co,ci,m,n]
 *   Y_l = phi(Z_l)          (phi = ReLU or identity)
 *
 * with zero padding of one cell, which for stride 1 is the output position
 * i - m + floor(k/2) of the paper's scatter equations (Eq. 1 and Eq. 2) read
 * in the gather direction (cross-correlation, as torch.conv2d), and for
 * stride 2 the usual PointPillars downsampling convolution.
 *
 * Storage is NHWC (a cell's channels are contiguous).  The loops follow the
 * definition: for each output cell, taps (m, n) in order, then input
 * channels; the innermost loop over output channels is left to the compiler's
 * auto-vectoriser.  Terms whose input value is exactly zero are skipped; they
 * contribute nothing to the sum.
 *
 * The bf16 storage variant rounds each layer's Y exactly like a bf16 map
 * written from an fp32 value: double -> float (round to nearest even, the C
 * conversion) -> bfloat16 (round to nearest even on the bit pattern).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_API __attribute__((visibility("default")))

/* Output extent of a 3x3 conv with zero padding 1 and stride s. */
static int out_extent(int n, int s) { return (n + 2 - 3) / s + 1; }

/*
 * Dense 3x3 convolution, zero padding 1.
 *   in  : [H][W][cin]   (NHWC, double)
 *   w   : [cout][cin][3][3] (OIHW, double)
 *   out : [Ho][Wo][cout], Ho = (H-1)/s + 1, Wo = (W-1)/s + 1
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
ORACLE_API int oracle_conv3x3_f64(const double* in, int H, int W, int cin,
                                  const double* w, int cout, int stride,
                                  double* out) {
    if (!in || !w || !out || H <= 0 || W <= 0 || cin <= 0 || cout <= 0 ||
        (stride != 1 && stride != 2))
        return -1;
    const int Ho = out_extent(H, stride), Wo = out_extent(W, stride);
    /* weights regrouped as [m][n][ci][co] so the inner loop runs over co */
    double* wt = (double*)malloc(sizeof(double) * 9u * (size_t)cin * (size_t)cout);
    if (!wt) return -1;
    for (int co = 0; co < cout; ++co)
        for (int ci = 0; ci < cin; ++ci)
            for (int m = 0; m < 3; ++m)
                for (int n = 0; n < 3; ++n)
                    wt[((size_t)(m * 3 + n) * cin + ci) * cout + co] =
                        w[(((size_t)co * cin + ci) * 3 + m) * 3 + n];

#pragma omp parallel for schedule(dynamic, 1)
    for (int y = 0; y < Ho; ++y) {
        for (int x = 0; x < Wo; ++x) {
            double* o = out + ((size_t)y * Wo + x) * cout;
            for (int co = 0; co < cout; ++co) o[co] = 0.0;
            for (int m = 0; m < 3; ++m) {
                const int iy = stride * y + m - 1;
                if (iy < 0 || iy >= H) continue;
                for (int n = 0; n < 3; ++n) {
                    const int ix = stride * x + n - 1;
                    if (ix < 0 || ix >= W) continue;
                    const double* a = in + ((size_t)iy * W + ix) * cin;
                    const double* wk = wt + (size_t)(m * 3 + n) * cin * cout;
                    for (int ci = 0; ci < cin; ++ci) {
                        const double v = a[ci];
                        if (v == 0.0) continue;
                        const double* wr = wk + (size_t)ci * cout;
                        for (int co = 0; co < cout; ++co) o[co] += v * wr[co];
                    }
                }
            }
        }
    }
    free(wt);
    return 0;
}

/* float -> bfloat16 bits, round to nearest even (finite inputs). */
static uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* In place: x <- (double) bf16( (float) x ). */
ORACLE_API void oracle_round_bf16(double* x, size_t n) {
    for (size_t i = 0; i < n; ++i) {
        const float f = (float)x[i];
        const uint32_t u = (uint32_t)f32_to_bf16_rne(f) << 16;
        float g;
        memcpy(&g, &u, 4);
        x[i] = (double)g;
    }
}

/*
 * The whole layer chain from scratch for one window.
 *   x0            : [H0][W0][C0] input canvas (exact values of the stored dtype)
 *   cin/cout/stride/relu : per-layer shape, L layers
 *   w[l]          : OIHW weights of layer l (exact values of the stored dtype)
 *   bf16_storage  : nonzero -> each Y_l is rounded as a bf16 map (see header)
 *   y[l]          : caller-allocated [H_l][W_l][cout_l] output, receives Y_l
 * Returns 0, or -1 on bad arguments / failure.
 */
ORACLE_API int oracle_backbone_f64(const double* x0, int H0, int W0, int C0, int L,
                                   const int* cin, const int* cout, const int* stride,
                                   const int* relu, const double* const* w,
                                   int bf16_storage, double* const* y) {
    if (!x0 || L <= 0 || !cin || !cout || !stride || !relu || !w || !y) return -1;
    const double* prev = x0;
    int H = H0, Wd = W0, C = C0;
    for (int l = 0; l < L; ++l) {
        if (cin[l] != C) return -1;
        if (oracle_conv3x3_f64(prev, H, Wd, C, w[l], cout[l], stride[l], y[l]) != 0) return -1;
        H = out_extent(H, stride[l]);
        Wd = out_extent(Wd, stride[l]);
        C = cout[l];
        const size_t n = (size_t)H * Wd * C;
        if (relu[l])
            for (size_t i = 0; i < n; ++i) y[l][i] = y[l][i] > 0.0 ? y[l][i] : 0.0;
        if (bf16_storage) oracle_round_bf16(y[l], n);
        prev = y[l];
    }
    return 0;
}

/*
 * Transposed convolution with kernel = stride s (the upsampling of the
 * PointPillars neck that brings every block to a common grid before the
 * concatenation; Sec. III-B, backbone paragraph, and Alg. 1, deconvolution
 * branch).  Kernel and stride equal, so every output cell has exactly one
 * input cell:
 *   out[s*i + a][s*j + b][co] = sum_ci in[i][j][ci] * w[ci][co][a][b]
 *   in  : [H][W][cin]; w: [cin][cout][s][s] (the PyTorch ConvTranspose2d
 *   layout); out : [H*s][W*s][cout].
 * Returns 0, or -1 on bad arguments.
 */
ORACLE_API int oracle_convT_f64(const double* in, int H, int W, int cin, const double* w, int cout, int s,
                                double* out) {
    if (!in || !w || !out || H <= 0 || W <= 0 || cin <= 0 || cout <= 0 || s <= 0) return -1;
    const int Wo = W * s;
#pragma omp parallel for schedule(dynamic, 1)
    for (int i = 0; i < H; ++i)
        for (int j = 0; j < W; ++j) {
            const double* a_in = in + ((size_t)i * W + j) * cin;
            for (int a = 0; a < s; ++a)
                for (int b = 0; b < s; ++b) {
                    double* o = out + ((size_t)(s * i + a) * Wo + (s * j + b)) * cout;
                    for (int co = 0; co < cout; ++co) o[co] = 0.0;
                    for (int ci = 0; ci < cin; ++ci) {
                        const double v = a_in[ci];
                        if (v == 0.0) continue;
                        const double* wr = w + (size_t)ci * cout * s * s;
                        for (int co = 0; co < cout; ++co) o[co] += v * wr[((size_t)co * s + a) * s + b];
                    }
                }
        }
    return 0;
}

#ifdef _OPENMP
#include <omp.h>
#endif
/* Threads the oracle's parallel loops use (OpenMP's current setting). */
ORACLE_API int oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
