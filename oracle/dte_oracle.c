/*
 * CPU oracle of the snapshot-free delta-extraction path -- TEST
 * INFRASTRUCTURE ONLY.  Only tests, the smoke check and the benchmark's
 * CPU-baseline leg may load this library; the product path never does.
 *
 * Plain, slow, obviously correct C: one element at a time, every floating
 * point operation a single IEEE binary32 operation with round-to-nearest-
 * even (built with gcc -ffp-contract=off, no fast-math, SSE arithmetic:
 * no fused multiply-add, subnormals kept, correctly rounded divide and
 * square root).  Shares no code with the HIP path.
 *
 * Operation order (the reading of the paper fixed for both sides): the step
 * scalars of the paper's AdamW inverse (sec. 4.1, eq. adamw_inverse) are
 * folded once, in binary64, into
 *     LRB1  = lr / (1 - beta1^t)        (step size with bias correction 1)
 *     RBC2  = 1 / (1 - beta2^t)         (reciprocal of bias correction 2)
 *     EPS   = eps
 *     DECAY = 1 - lr * weight_decay     (multiplicative decoupled decay)
 * each rounded once to binary32.  Then per element
 *     u  = (LRB1 * m) / (sqrt(v * RBC2) + EPS)
 *     forward (appendix A, eq. appendix_adamw_forward):   p  = DECAY * p_prev - u
 *     inverse (sec. 4.1, eq. adamw_inverse):              ph = (p + u) / DECAY
 * which is the paper's expression with the bias corrections folded into
 * the two scalars, evaluated left to right.
 *
 * Literal order (order = 1): eq. adamw_inverse operation by operation, with
 * LR = lr, BC1 = 1 - beta1^t, BC2 = 1 - beta2^t rounded once to binary32:
 *     u  = LR * ((m / BC1) / (sqrt(v / BC2) + EPS))
 * (four divisions with the one by DECAY), used by the forward step and the
 * inverse alike.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

typedef struct {
    float lrb1, rbc2, eps, decay;   /* inverse and forward */
    float b1, b2, omb1, omb2;       /* forward moment update only */
    float lr, bc1, bc2;             /* literal order */
    int32_t order;                  /* 0: folded, 1: literal */
} oracle_scalars;

/* Step scalars (sec. 4.1, eq. adamw_inverse; appendix A): binary64 math,
 * one rounding to binary32 each.  Returns 0, or -1 on invalid input. */
int oracle_derive_scalars(double lr, double beta1, double beta2, double eps, double wd,
                          int64_t step, int32_t order, oracle_scalars* out)
{
    if (step < 1 || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) ||
        (order != 0 && order != 1))
        return -1;
    const double bc1 = 1.0 - pow(beta1, (double)step);
    const double bc2 = 1.0 - pow(beta2, (double)step);
    const double decay = 1.0 - lr * wd;
    if (!(decay > 0.0) || !(bc1 > 0.0) || !(bc2 > 0.0)) return -1;
    out->lrb1 = (float)(lr / bc1);
    out->rbc2 = (float)(1.0 / bc2);
    out->eps = (float)eps;
    out->decay = (float)decay;
    out->b1 = (float)beta1;
    out->b2 = (float)beta2;
    out->omb1 = (float)(1.0 - beta1);
    out->omb2 = (float)(1.0 - beta2);
    out->lr = (float)lr;
    out->bc1 = (float)bc1;
    out->bc2 = (float)bc2;
    out->order = order;
    return 0;
}

/* Adaptive step term u = (LRB1*m) / (sqrt(v*RBC2) + EPS), one element
 * (literal order: LR * ((m / BC1) / (sqrt(v / BC2) + EPS))). */
static float oracle_step_term(float m, float v, const oracle_scalars* s)
{
    if (s->order == 1) {
        const float mh = m / s->bc1;   /* m_t / (1 - beta1^t)         */
        const float vq = v / s->bc2;   /* v_t / (1 - beta2^t)         */
        const float sq = sqrtf(vq);
        const float d = sq + s->eps;
        const float r = mh / d;
        return s->lr * r;              /* eta_t times the ratio       */
    }
    const float vh = v * s->rbc2;      /* v / (1 - beta2^t)           */
    const float sq = sqrtf(vh);        /* sqrt of the corrected moment */
    const float den = sq + s->eps;     /* + epsilon                    */
    const float num = s->lrb1 * m;     /* lr * m / (1 - beta1^t)       */
    return num / den;
}

/* One forward AdamW step (sec. 4.1, eq. adamw_moments; appendix A,
 * eq. appendix_adamw_forward), producing the post-step state the method
 * reads.  Element-wise over n elements. */
void oracle_adamw_forward(const float* p_prev, const float* m_prev, const float* v_prev,
                          const float* g, int64_t n, const oracle_scalars* s, float* p,
                          float* m, float* v)
{
    for (int64_t i = 0; i < n; ++i) {
        const float gi = g[i];
        const float m1 = s->b1 * m_prev[i];
        const float m2 = s->omb1 * gi;
        const float mt = m1 + m2;                 /* m_t = b1 m_{t-1} + (1-b1) g   */
        const float g2 = gi * gi;
        const float v1 = s->b2 * v_prev[i];
        const float v2 = s->omb2 * g2;
        const float vt = v1 + v2;                 /* v_t = b2 v_{t-1} + (1-b2) g^2 */
        const float u = oracle_step_term(mt, vt, s);
        const float a = s->decay * p_prev[i];     /* (1 - lr wd) theta_{t-1}       */
        p[i] = a - u;
        m[i] = mt;
        v[i] = vt;
    }
}

/* AdamW inversion (sec. 4.1, eq. adamw_inverse): theta_hat_{t-1} per
 * element from theta_t, m_t, v_t. */
void oracle_invert(const float* p, const float* m, const float* v, int64_t n,
                   const oracle_scalars* s, float* p_hat)
{
    for (int64_t i = 0; i < n; ++i) {
        const float u = oracle_step_term(m[i], v[i], s);
        const float num = p[i] + u;
        p_hat[i] = num / s->decay;
    }
}

/* BF16 quantisation Q_BF16 of sec. 4.2.1, as round-to-nearest-even of the
 * binary32 bit pattern: keep the upper 16 bits after adding half an ulp of
 * BF16 (0x7FFF) plus the parity of the kept part, so exact ties go to the
 * even pattern; overflow carries into +-inf; subnormals are kept.  Any NaN
 * becomes the canonical quiet NaN 0x7FC0. */
uint16_t oracle_bf16(float x)
{
    if (x != x) return (uint16_t)0x7FC0u;
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    const uint64_t r = (uint64_t)u + 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(r >> 16);
}

void oracle_bf16_array(const float* x, int64_t n, uint16_t* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16(x[i]);
}

/* BF16 of every binary32 pattern in [first, first + n) (for the exhaustive
 * check of the rounding rule). */
void oracle_bf16_patterns(uint32_t first, int64_t n, uint16_t* out)
{
    for (int64_t i = 0; i < n; ++i) {
        const uint32_t u = first + (uint32_t)i;
        float x;
        memcpy(&x, &u, sizeof x);
        out[i] = oracle_bf16(x);
    }
}
