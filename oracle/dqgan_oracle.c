/*
 * DQGAN oracle: a plain, slow, scalar CPU implementation of one iteration of
 * the distributed optimistic-mirror-descent loop with error feedback and a
 * delta-approximate compressor (Algorithm 2 of Chen, Yang, Shen, Pang,
 * "A Distributed Training Algorithm of Generative Adversarial Networks with
 * Quantized Gradients", arXiv:2010.13359).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's library.  It shares no
 * code, header, table or constant generator with the GPU library, and the GPU
 * library never calls it.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared.
 * Every float operation below is one IEEE-754 binary32 operation with
 * round-to-nearest-even, unless the comment says double.  No FMA contraction.
 *
 * Readings of points the paper leaves open (each is listed with its reason in
 * the design notes):
 *   - p = fl(fl(eta*g) + e): two roundings, no fused multiply-add.
 *   - Segment scales: the sums are taken in double in ascending index order
 *     and rounded once to binary32.
 *   - Scaled sign: scale = ||p_seg||_1 / n_seg; the code is the IEEE sign bit,
 *     so +0 maps to +scale and -0 to -scale.
 *   - s-level stochastic quantizer: r = fl(|p| * fl(s/sigma)),
 *     l = min(floor(r), s), frac = r - l, round up iff u < frac, level capped
 *     at s; the decoded value is copysign(fl(level * fl(sigma/s)), p).
 *     For sigma < 2^-64 both |p| and sigma are first multiplied by 2^64
 *     (exact) and the decoded magnitude by 2^-64 (one rounding), so that
 *     fl(s/sigma) cannot overflow and fl(sigma/s) keeps its significand;
 *     wherever the plain evaluation stays in the normal range the two give
 *     the same bits.  A segment whose norm is 0 or not finite (a norm that
 *     the binary32 scale of the message cannot hold) quantizes to level 0
 *     everywhere, and so does a zero element (|v_i| / ||v|| = 0 gives l = 0
 *     and round-up probability 0).
 *   - Uniforms for stochastic rounding come from Philox4x32-10 with key
 *     (lo32(seed), hi32(seed)) and counter (lo32(i>>2), m, t, hi32(i>>2));
 *     element i takes output word (i & 3) and u = (word >> 8) * 2^-24.
 *   - Top-k keeps the k largest |p| with ties broken towards the lower index,
 *     and transmits (value, index) pairs in ascending index order.
 *   - Aggregation sums the M decoded messages in ascending worker order in
 *     binary32 and divides the sum by M once.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Counter-based generator: Philox4x32 with 10 rounds (Salmon, Moraes, Dror,
 * Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11).  Each round
 * multiplies counter words 0 and 2 by the two round multipliers, producing
 * 64-bit products; the new counter is (hi(c2*M1) ^ c1 ^ k0, lo(c2*M1),
 * hi(c0*M0) ^ c3 ^ k1, lo(c0*M0)).  The key is advanced by the two Weyl
 * increments between rounds. */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t prod0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
        uint64_t prod1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
        uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The uniform in [0,1) used to round element i of worker m at iteration t. */
float oracle_uniform(uint64_t seed, int64_t i, int32_t m, uint32_t t) {
    uint64_t block = (uint64_t)i >> 2;
    uint32_t ctr[4] = {(uint32_t)block, (uint32_t)m, t, (uint32_t)(block >> 32)};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    uint32_t word = out[i & 3];
    return (float)(word >> 8) * 0x1.0p-24f;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 2, worker side: p_t = eta * F(w_{t-1/2}) + e_{t-1}. */
void oracle_ef_accumulate(int64_t n, float eta, const float *g, const float *e, float *p) {
    for (int64_t i = 0; i < n; ++i) {
        float eg = eta * g[i];
        p[i] = eg + e[i];
    }
}

/* Scale of the scaled-sign compressor: the mean magnitude ||p||_1 / n. */
float oracle_scale_l1mean(int64_t n, const float *p) {
    double sum = 0.0;
    for (int64_t i = 0; i < n; ++i) sum += fabs((double)p[i]);
    return (float)(sum / (double)n);
}

/* ||p||_2 of the stochastic quantizer (equation qsgd). */
float oracle_scale_l2(int64_t n, const float *p) {
    double sum = 0.0;
    for (int64_t i = 0; i < n; ++i) sum += (double)p[i] * (double)p[i];
    return (float)sqrt(sum);
}

/* ||p||_inf, the variant that replaces the 2-norm (Section 2.4, Appendix A). */
float oracle_scale_linf(int64_t n, const float *p) {
    float mx = 0.0f;
    for (int64_t i = 0; i < n; ++i) {
        float a = fabsf(p[i]);
        if (a > mx) mx = a;
    }
    return mx;
}

/* Scaled sign: phat_i = +scale if the sign bit of p_i is clear, -scale
 * otherwise; e_i = p_i - phat_i.  bits[i] receives the sign bit (1 = minus). */
void oracle_sign_encode(int64_t n, const float *p, float scale, uint8_t *bits, float *phat, float *e_out) {
    for (int64_t i = 0; i < n; ++i) {
        int neg = signbit(p[i]) ? 1 : 0;
        float q = neg ? -scale : scale;
        bits[i] = (uint8_t)neg;
        phat[i] = q;
        e_out[i] = p[i] - q;
    }
}

/* The range in which equation (qsgd) is evaluated for a segment of norm
 * sigma.  r = |v_i| s / sigma does not change when v is scaled, but
 * fl(s/sigma) overflows binary32 once sigma < s / FLT_MAX and fl(sigma/s)
 * drops significand bits once it is subnormal.  For sigma < 2^-64 the
 * magnitudes and the norm are multiplied by up = 2^64 (exact: every |v_i| is
 * at most about sigma) and the decoded magnitude by down = 2^-64.  Returns 0
 * for a norm of 0 or one that is not finite: nothing of the segment is sent. */
static int qsgd_range(float sigma, float *up, float *down) {
    if (!(sigma > 0.0f) || !(sigma <= FLT_MAX)) return 0;
    if (sigma < 0x1.0p-64f) {
        *up = 0x1.0p64f;
        *down = 0x1.0p-64f;
    } else {
        *up = 1.0f;
        *down = 1.0f;
    }
    return 1;
}

/* s-level stochastic quantizer (equation qsgd): for the segment starting at
 * row index i0, xi_i = l/s or (l+1)/s with P[(l+1)/s] = |p_i| s / sigma - l.
 * levels[i] receives the integer level, bits[i] the sign bit. */
void oracle_qsgd_encode(int64_t n, int64_t i0, const float *p, float sigma, int32_t s,
                        uint64_t seed, int32_t m, uint32_t t,
                        uint8_t *bits, uint16_t *levels, float *phat, float *e_out) {
    float fs = (float)s;
    float up = 1.0f, down = 1.0f, inv = 0.0f, step = 0.0f;
    int live = qsgd_range(sigma, &up, &down);
    if (live) {
        float su = sigma * up;
        inv = fs / su;
        step = su / fs;
    }
    for (int64_t i = 0; i < n; ++i) {
        int neg = signbit(p[i]) ? 1 : 0;
        int32_t level = 0;
        float a = fabsf(p[i]);
        if (live && a > 0.0f) {
            float r = (a * up) * inv;
            float l = floorf(r);
            if (l > fs) l = fs;
            float frac = (l == fs) ? 0.0f : r - l;
            float u = oracle_uniform(seed, i0 + i, m, t);
            level = (int32_t)l + ((u < frac) ? 1 : 0);
            if (level > s) level = s;
        }
        float mag = ((float)level * step) * down;
        float q = copysignf(mag, p[i]);
        bits[i] = (uint8_t)neg;
        levels[i] = (uint16_t)level;
        phat[i] = q;
        e_out[i] = p[i] - q;
    }
}

/* Top-k (k-contraction, Theorem 1): keep the k entries of largest magnitude,
 * ties to the lower index.  The selection is the first k entries of the list
 * ordered by (|p| descending, index ascending); the magnitude order is the
 * order of the binary32 bit patterns of |p|. */
typedef struct { uint32_t key; int64_t idx; } topk_item;

static int topk_cmp(const void *a, const void *b) {
    const topk_item *x = (const topk_item *)a, *y = (const topk_item *)b;
    if (x->key != y->key) return (x->key > y->key) ? -1 : 1;
    if (x->idx != y->idx) return (x->idx < y->idx) ? -1 : 1;
    return 0;
}
static int idx_cmp(const void *a, const void *b) {
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return (x < y) ? -1 : (x > y) ? 1 : 0;
}

static uint32_t magnitude_key(float v) {
    float a = fabsf(v);
    uint32_t k;
    memcpy(&k, &a, sizeof k);
    return k;
}

/* Returns 0 on success, -1 if scratch memory could not be obtained. */
int oracle_topk(int64_t d, int64_t k, const float *p, uint32_t *idx, float *val, float *phat, float *e_out) {
    topk_item *items = (topk_item *)malloc((size_t)d * sizeof(topk_item));
    if (!items) return -1;
    for (int64_t i = 0; i < d; ++i) {
        items[i].key = magnitude_key(p[i]);
        items[i].idx = i;
    }
    qsort(items, (size_t)d, sizeof(topk_item), topk_cmp);
    for (int64_t j = 0; j < k; ++j) idx[j] = (uint32_t)items[j].idx;
    free(items);
    qsort(idx, (size_t)k, sizeof(uint32_t), idx_cmp);
    for (int64_t i = 0; i < d; ++i) {
        phat[i] = 0.0f;
        e_out[i] = p[i] - 0.0f;
    }
    for (int64_t j = 0; j < k; ++j) {
        int64_t i = idx[j];
        val[j] = p[i];
        phat[i] = p[i];
        e_out[i] = p[i] - p[i];
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The message format.  Sign plane: element i of a row is bit (i & 31) of word
 * i >> 5.  Level plane with b bits per element (b = 8 or 4): element i is the
 * b-bit field starting at bit b*(i mod 32/b) of word i / (32/b).  Bits beyond
 * the last element of a row are zero. */
void oracle_pack_bits(int64_t n, int32_t b, const uint16_t *fields, uint32_t *words, int64_t nwords) {
    int64_t per = 32 / b;
    for (int64_t w = 0; w < nwords; ++w) words[w] = 0u;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t f = (uint32_t)fields[i] & ((b == 32) ? 0xFFFFFFFFu : ((1u << b) - 1u));
        words[i / per] |= f << (uint32_t)(b * (i % per));
    }
}

void oracle_unpack_bits(int64_t n, int32_t b, const uint32_t *words, uint16_t *fields) {
    int64_t per = 32 / b;
    uint32_t mask = (1u << b) - 1u;
    for (int64_t i = 0; i < n; ++i)
        fields[i] = (uint16_t)((words[i / per] >> (uint32_t)(b * (i % per))) & mask);
}

/* Decoding the message of one segment back to phat (what the server does
 * after pulling it).  kind 0 = scaled sign, 1 = s-level quantizer. */
void oracle_decode_segment(int32_t kind, int64_t n, const uint16_t *signs, const uint16_t *levels,
                           float scale, int32_t s, float *phat) {
    float up = 1.0f, down = 1.0f, step = 0.0f;
    if (kind == 1 && qsgd_range(scale, &up, &down)) step = (scale * up) / (float)s;
    for (int64_t i = 0; i < n; ++i) {
        if (kind == 0) {
            phat[i] = signs[i] ? -scale : scale;
        } else {
            float mag = ((float)levels[i] * step) * down;
            phat[i] = signs[i] ? -mag : mag;
        }
    }
}

/* The m-bit code of Appendix A: q(v_i, s) takes one of the 2k+1 values
 * -B_k .. B_k with k = 2^(m-1) - 1, which m bits hold as sign and magnitude:
 * bit m-1 is the sign, bits 0..m-2 the level r (reading: B_r = r / k, so that
 * the rounding rule is the one of equation (qsgd) with k levels). */
void oracle_mbit_fields(int64_t n, int32_t mbits, const uint8_t *bits, const uint16_t *levels, uint16_t *fields) {
    for (int64_t i = 0; i < n; ++i)
        fields[i] = (uint16_t)(((uint32_t)bits[i] << (mbits - 1)) | levels[i]);
}

void oracle_mbit_split(int64_t n, int32_t mbits, const uint16_t *fields, uint16_t *signs, uint16_t *levels) {
    uint16_t mask = (uint16_t)((1u << (mbits - 1)) - 1u);
    for (int64_t i = 0; i < n; ++i) {
        signs[i] = (uint16_t)(fields[i] >> (mbits - 1));
        levels[i] = (uint16_t)(fields[i] & mask);
    }
}

/* ------------------------------------------------------------------------ */
/* Server: qhat = (1/M) sum_m phat^(m) (Algorithm 2).  The running sum S
 * starts at phat^(0) and adds phat^(1), ..., phat^(M-1) in that order. */
void oracle_aggregate(int32_t M, int64_t d, int64_t ld, const float *phat, float *qhat) {
    for (int64_t i = 0; i < d; ++i) {
        float S = phat[i];
        for (int32_t m = 1; m < M; ++m) S = S + phat[(int64_t)m * ld + i];
        qhat[i] = S / (float)M;
    }
}

/* Worker: w_t = w_{t-1} - qhat_t (Algorithm 2, last worker step). */
void oracle_omd_update(int64_t d, const float *qhat, float *w) {
    for (int64_t i = 0; i < d; ++i) w[i] = w[i] - qhat[i];
}

/* Worker: the next evaluation point w_{t+1/2} = w_t - (eta F(w_{t-1/2}) + e_t)
 * (Algorithm 2, first worker step of iteration t+1, which reuses the stored
 * gradient and compensates the error a second time). */
void oracle_extrapolate(int64_t d, float eta, const float *w, const float *g, const float *e, float *wx) {
    for (int64_t i = 0; i < d; ++i) {
        float eg = eta * g[i];
        float x = eg + e[i];
        wx[i] = w[i] - x;
    }
}

/* ------------------------------------------------------------------------ */
/* One full iteration over M workers (rows of stride ld) for the compressor
 * `kind` (0 sign, 1 s-level quantizer, 2 top-k, 3 identity, 4 the m-bit
 * sign-magnitude quantizer of Appendix A with `levels` = m bits).
 *
 * In: G (the fresh gradients), E (e_{t-1}), W (w_{t-1}).
 * Out: E (e_t), W (w_t), WX (next evaluation points), the message planes and
 * qhat.  If scales_in is non-NULL the segment scales are taken from it (the
 * teacher-forced comparison) instead of being computed.
 * For the identity compressor the message is the dense phat in val[M][ld].
 * Returns 0, or -1 when a scratch allocation fails or an argument is invalid. */
typedef struct {
    int64_t d, ld;
    int32_t M, n_seg;
    const int64_t *seg_offsets;  /* n_seg + 1 entries, 0 ... d */
    int32_t kind, norm;          /* norm: 1 = L1 mean, 2 = L2, 3 = Linf */
    int32_t levels;              /* s of the quantizer */
    int64_t k;
    uint64_t seed;
} oracle_desc;

int oracle_step(const oracle_desc *D, float eta, uint32_t t, const float *G, float *E, float *W, float *WX,
                uint32_t *sign_words, uint32_t *level_words, float *scales, float *val, uint32_t *idx,
                float *qhat, const float *scales_in) {
    int64_t d = D->d, ld = D->ld;
    int32_t M = D->M;
    if (d < 1 || ld < d || M < 1) return -1;
    int32_t bits_per_level = (D->levels == 255) ? 8 : (D->levels == 15) ? 4 : 0;
    int32_t mbits = (D->kind == 4) ? D->levels : 0;           /* Appendix A: m bits per code */
    int32_t mlevels = mbits ? (1 << (mbits - 1)) - 1 : 0;     /* k = 2^(m-1) - 1 */
    float *p = (float *)malloc((size_t)d * sizeof(float));
    float *phat = (float *)malloc((size_t)d * sizeof(float));
    float *dec = (float *)malloc((size_t)d * sizeof(float));
    float *S = (float *)malloc((size_t)d * sizeof(float));
    uint8_t *bits = (uint8_t *)malloc((size_t)d);
    uint16_t *lv = (uint16_t *)malloc((size_t)d * sizeof(uint16_t));
    uint16_t *fs = (uint16_t *)malloc((size_t)d * sizeof(uint16_t));
    uint16_t *fl = (uint16_t *)malloc((size_t)d * sizeof(uint16_t));
    int rc = 0;
    if (!p || !phat || !dec || !S || !bits || !lv || !fs || !fl) { rc = -1; goto done; }

    for (int32_t m = 0; m < M; ++m) {
        const float *g = G + (int64_t)m * ld;
        float *e = E + (int64_t)m * ld;
        oracle_ef_accumulate(d, eta, g, e, p);
        if (D->kind == 0 || D->kind == 1) {
            for (int32_t j = 0; j < D->n_seg; ++j) {
                int64_t a = D->seg_offsets[j], b = D->seg_offsets[j + 1];
                int64_t n = b - a;
                float sc;
                if (scales_in) sc = scales_in[(int64_t)m * D->n_seg + j];
                else if (D->kind == 0) sc = oracle_scale_l1mean(n, p + a);
                else if (D->norm == 3) sc = oracle_scale_linf(n, p + a);
                else sc = oracle_scale_l2(n, p + a);
                scales[(int64_t)m * D->n_seg + j] = sc;
                if (D->kind == 0) {
                    oracle_sign_encode(n, p + a, sc, bits + a, phat + a, e + a);
                    for (int64_t i = a; i < b; ++i) lv[i] = 0;
                } else {
                    oracle_qsgd_encode(n, a, p + a, sc, D->levels, D->seed, m, t, bits + a, lv + a, phat + a, e + a);
                }
            }
            /* push: pack the sign plane (and level plane) of this worker */
            for (int64_t i = 0; i < d; ++i) fs[i] = bits[i];
            oracle_pack_bits(d, 1, fs, sign_words + (int64_t)m * (ld / 32), ld / 32);
            if (D->kind == 1)
                oracle_pack_bits(d, bits_per_level, lv, level_words + (int64_t)m * (ld * bits_per_level / 32),
                                 ld * bits_per_level / 32);
            /* pull: the server decodes the message it received */
            oracle_unpack_bits(d, 1, sign_words + (int64_t)m * (ld / 32), fs);
            if (D->kind == 1)
                oracle_unpack_bits(d, bits_per_level, level_words + (int64_t)m * (ld * bits_per_level / 32), fl);
            for (int32_t j = 0; j < D->n_seg; ++j) {
                int64_t a = D->seg_offsets[j], b = D->seg_offsets[j + 1];
                oracle_decode_segment(D->kind, b - a, fs + a, fl + a, scales[(int64_t)m * D->n_seg + j],
                                      D->levels, dec + a);
            }
        } else if (D->kind == 4) {
            int64_t rw = ld * mbits / 32;  /* code words per row */
            for (int32_t j = 0; j < D->n_seg; ++j) {
                int64_t a = D->seg_offsets[j], b = D->seg_offsets[j + 1];
                int64_t n = b - a;
                float sc;
                if (scales_in) sc = scales_in[(int64_t)m * D->n_seg + j];
                else if (D->norm == 3) sc = oracle_scale_linf(n, p + a);
                else sc = oracle_scale_l2(n, p + a);
                scales[(int64_t)m * D->n_seg + j] = sc;
                oracle_qsgd_encode(n, a, p + a, sc, mlevels, D->seed, m, t, bits + a, lv + a, phat + a, e + a);
            }
            /* push: one m-bit sign-magnitude code per element */
            oracle_mbit_fields(d, mbits, bits, lv, fs);
            oracle_pack_bits(d, mbits, fs, level_words + (int64_t)m * rw, rw);
            /* pull: the server splits and decodes the codes */
            oracle_unpack_bits(d, mbits, level_words + (int64_t)m * rw, fl);
            oracle_mbit_split(d, mbits, fl, fs, lv);
            for (int32_t j = 0; j < D->n_seg; ++j) {
                int64_t a = D->seg_offsets[j], b = D->seg_offsets[j + 1];
                oracle_decode_segment(1, b - a, fs + a, lv + a, scales[(int64_t)m * D->n_seg + j], mlevels, dec + a);
            }
        } else if (D->kind == 2) {
            if (oracle_topk(d, D->k, p, idx + (int64_t)m * D->k, val + (int64_t)m * D->k, phat, e) != 0) {
                rc = -1; goto done;
            }
            for (int64_t i = 0; i < d; ++i) dec[i] = 0.0f;
            for (int64_t j = 0; j < D->k; ++j) {
                int64_t i = idx[(int64_t)m * D->k + j];
                dec[i] = val[(int64_t)m * D->k + j];
            }
        } else {
            for (int64_t i = 0; i < d; ++i) {
                val[(int64_t)m * ld + i] = p[i];
                e[i] = p[i] - p[i];
                dec[i] = val[(int64_t)m * ld + i];
            }
        }
        /* server running sum, ascending m (the same per-element order as
         * oracle_aggregate, with the loops over m and i swapped) */
        if (m == 0) for (int64_t i = 0; i < d; ++i) S[i] = dec[i];
        else for (int64_t i = 0; i < d; ++i) S[i] = S[i] + dec[i];
    }
    for (int64_t i = 0; i < d; ++i) qhat[i] = S[i] / (float)M;
    oracle_omd_update(d, qhat, W);
    for (int32_t m = 0; m < M; ++m)
        oracle_extrapolate(d, eta, W, G + (int64_t)m * ld, E + (int64_t)m * ld, WX + (int64_t)m * ld);
done:
    free(p); free(phat); free(dec); free(S); free(bits); free(lv); free(fs); free(fl);
    return rc;
}
