/*
 * CPU oracle for the sparse INT8 linear layer -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg load this
 * file's library. It is the plain definition of what the accelerated path
 * computes, written for a reader to check by eye. It never sees a packed or
 * compressed weight: it multiplies by the dense int8 weight, zeros included,
 * because the block-sparse kernel of the paper (Section "Sparse GEMM
 * operators", Algorithm 1, Figure 1) reaches exactly the dense product -- the
 * zero blocks it skips contribute nothing to an integer sum.
 *
 * Shares no code, header or constant generator with the HIP library.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (no fast-math), so
 * every fp32 operation below is one separately rounded IEEE operation in the
 * order written.
 *
 * Conventions: X [M x K] int8 row-major (tokens x input features),
 * W [N x K] int8 row-major (output x input features), Y [M x N] row-major.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum {
    ORACLE_ACC_I32 = 0,  /* raw int32 accumulators                       */
    ORACLE_F32 = 1,      /* dequant + bias -> fp32                        */
    ORACLE_F32_GELU = 2, /* dequant + bias + GELU(erf) -> fp32            */
    ORACLE_I8 = 3,       /* dequant + bias, requantise -> int8            */
    ORACLE_I8_GELU = 4   /* dequant + bias + GELU(erf), requantise -> int8 */
};

/*
 * Step 1 -- the contraction. Section "Sparse GEMM operators": the kernel
 * multiplies the dense (quantised) input by the block-sparse weight; with
 * VNNI (int8 x int8 -> int32 dot products, Algorithm 1) the accumulation is
 * exact integer arithmetic. acc[m][n] = sum_k X[m][k] * W[n][k], k ascending.
 * |acc| <= 127*127*K, below 2^31 for K <= 133143, so int32 never overflows at
 * the sizes this library accepts.
 */
static int32_t dot_row(const int8_t *x, const int8_t *w, int32_t k)
{
    int32_t acc = 0;
    for (int32_t i = 0; i < k; ++i)
        acc += (int32_t)x[i] * (int32_t)w[i];
    return acc;
}

void oracle_acc(const int8_t *x, const int8_t *w, int64_t m, int32_t n, int32_t k, int32_t *acc)
{
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < m; ++r)
        for (int32_t c = 0; c < n; ++c)
            acc[r * n + c] = dot_row(x + r * (int64_t)k, w + (int64_t)c * k, k);
}

/*
 * Step 2 -- GELU, exact (erf) form: GELU(y) = y * Phi(y)
 *         = 0.5 * y * (1 + erf(y / sqrt 2)).
 * The graph optimisation (Appendix "Graph optimization") fuses the
 * post-operators that follow an InnerProduct into it; the FFN's first linear
 * is followed by GELU in DistilBERT. Evaluated in fp32 in this order:
 *   t = y * fl(1/sqrt 2);  e = erff(t);  g = (0.5 * y) * (1 + e).
 */
float oracle_gelu(float y)
{
    float t = y * 0.70710678118654752f;
    float e = erff(t);
    float h = 0.5f * y;
    float one_e = 1.0f + e;
    return h * one_e;
}

/*
 * Step 3 -- requantisation ("downconvert", Algorithm 1 and Section "Sparse
 * GEMM operators"): symmetric int8 with per-tensor scale so and zero point 0:
 *   q = clamp(rint(g * fl(1/so)), -127, 127), rint = round half to even.
 */
static int8_t requant(float g, float inv_so)
{
    float v = g * inv_so;
    float r = rintf(v);
    if (r > 127.0f) r = 127.0f;
    if (r < -127.0f) r = -127.0f;
    return (int8_t)r;
}

/*
 * The fused epilogue (Section "Sparse GEMM operators": the intermediate int32
 * output plus bias C gives the final output; Appendix "Graph optimization":
 * post-operators fused into the InnerProduct). Per element, fp32, in order:
 *   s = sx * sw[n];  y = (float)acc * s;  y = y + b[n];
 *   [g = GELU(y)];   [q = requant(g, so)].
 */
static void epilogue_one(int32_t a, int32_t c, float sx, const float *sw, const float *bias,
                         int32_t kind, float inv_so, void *out, int64_t i)
{
    if (kind == ORACLE_ACC_I32) {
        ((int32_t *)out)[i] = a;
        return;
    }
    float s = sx * sw[c];
    float y = (float)a * s;
    y = y + (bias ? bias[c] : 0.0f);
    float g = (kind == ORACLE_F32_GELU || kind == ORACLE_I8_GELU) ? oracle_gelu(y) : y;
    if (kind == ORACLE_F32 || kind == ORACLE_F32_GELU)
        ((float *)out)[i] = g;
    else
        ((int8_t *)out)[i] = requant(g, inv_so);
}

void oracle_epilogue(const int32_t *acc, int64_t m, int32_t n, float sx, const float *sw,
                     const float *bias, int32_t kind, float so, void *out)
{
    float inv_so = 1.0f / so;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < m; ++r)
        for (int32_t c = 0; c < n; ++c)
            epilogue_one(acc[r * n + c], c, sx, sw, bias, kind, inv_so, out, r * n + c);
}

/* The whole layer for a block of rows: contraction, then the epilogue.
 * Rows are independent, so the caller may pass any subset of tokens. */
void oracle_linear(const int8_t *x, const int8_t *w, int64_t m, int32_t n, int32_t k, float sx,
                   const float *sw, const float *bias, int32_t kind, float so, void *out)
{
    float inv_so = 1.0f / so;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t r = 0; r < m; ++r)
        for (int32_t c = 0; c < n; ++c)
            epilogue_one(dot_row(x + r * (int64_t)k, w + (int64_t)c * k, k), c, sx, sw, bias, kind,
                         inv_so, out, r * n + c);
}

/*
 * Activation quantisation for the first op of a chain (Section
 * "Post-training quantization": INT8 with calibrated scales): symmetric
 * per-tensor, q = clamp(rint(x * fl(1/s)), -127, 127). Inputs must be finite.
 */
void oracle_quantize(const float *x, int64_t count, float scale, int8_t *q)
{
    float inv = 1.0f / scale;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        q[i] = requant(x[i], inv);
}

/* max |v| over a buffer, for calibrating an output scale so = max|g| / 127. */
float oracle_absmax_f32(const float *v, int64_t count)
{
    float best = 0.0f;
    for (int64_t i = 0; i < count; ++i) {
        float a = fabsf(v[i]);
        if (a > best) best = a;
    }
    return best;
}

/* Threads for the OpenMP loops above (timing only; results do not depend on it). */
void oracle_set_threads(int n)
{
    if (n > 0) omp_set_num_threads(n);
}

/* Number of threads the OpenMP loops above use. */
int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
