/*
 * Seeded synthetic-input generator shared by the CPU oracle and the GPU path.
 *
 * It holds none of the decoder's arithmetic: it only turns (seed, stream,
 * element index) into numbers and stores them in a requested storage type.
 *
 * Uniform bits come from Philox4x32-10, the counter-based generator of
 * Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3"
 * (SC'11): a 128-bit counter and a 64-bit key go through ten rounds of two
 * 32x32->64 multiplies, with the key bumped by two Weyl constants between
 * rounds.  Normal draws use the Box-Muller transform (Box and Muller, 1958).
 *
 * Element i of a stream uses Philox block i/4 with counter
 * (block_lo, block_hi, stream_lo, stream_hi) and key (seed_lo, seed_hi).
 * A block yields four words x0..x3; the pairs (x0,x1) and (x2,x3) each give
 * two normals: r = sqrt(-2 ln u1), u1 = (x_even + 0.5) 2^-32, angle
 * 2 pi x_odd 2^-32, first cos then sin.  ln, cos and sin are evaluated by the
 * series below rather than libm, so the draws do not depend on the host's
 * math library.  The draw is computed in double,
 * mean + std * n, and rounded once to float (round to nearest even).  The
 * fp16 and bf16 outputs are the round-to-nearest-even conversion of that
 * float draw.
 *
 * Everything is compiled with -ffp-contract=off so the sequence of roundings
 * is the one written here on any IEEE-754 host.
 */
#include <math.h> /* sqrt only */
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox_round(uint32_t c[4], const uint32_t k[2]) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
    uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c[1] ^ k[0];
    uint32_t n2 = hi0 ^ c[3] ^ k[1];
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
}

/* Philox4x32 with R rounds; exported for known-answer tests. */
void synth_philox4x32(const uint32_t ctr_in[4], const uint32_t key_in[2], int rounds,
                      uint32_t out[4]) {
    uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    uint32_t k[2] = {key_in[0], key_in[1]};
    for (int r = 0; r < rounds; ++r) {
        if (r > 0) {
            k[0] += PHILOX_W0;
            k[1] += PHILOX_W1;
        }
        philox_round(c, k);
    }
    memcpy(out, c, sizeof(c));
}

static inline void philox_block(uint64_t seed, uint64_t stream, uint64_t block, uint32_t out[4]) {
    uint32_t c[4] = {(uint32_t)block, (uint32_t)(block >> 32), (uint32_t)stream,
                     (uint32_t)(stream >> 32)};
    uint32_t k[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    synth_philox4x32(c, k, 10, out);
}

static const double LN2 = 0.69314718055994530941723212145818;
static const double HALF_PI = 1.5707963267948966192313216916398;
static const double INV_2_32 = 2.3283064365386962890625e-10; /* 2^-32 */

/*
 * Natural log of u in (0, 1] from its definition: u = m 2^e with m in
 * [sqrt(1/2), sqrt(2)), ln u = e ln 2 + 2 atanh(t), t = (m - 1)/(m + 1),
 * atanh t = t + t^3/3 + t^5/5 + ...; |t| <= 0.1716, so terms through t^19
 * leave a truncation error below 1e-16.  Only + - * / are used, so the
 * result is the same on every IEEE-754 host.
 */
static inline double ln_unit(double u) {
    uint64_t b;
    memcpy(&b, &u, 8);
    int e = (int)((b >> 52) & 0x7FF) - 1023;
    uint64_t mb = (b & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull; /* m in [1, 2) */
    double m;
    memcpy(&m, &mb, 8);
    if (m > 1.4142135623730950488) {
        m *= 0.5;
        e += 1;
    }
    double t = (m - 1.0) / (m + 1.0);
    double t2 = t * t;
    double s = 1.0 / 19.0;
    s = s * t2 + 1.0 / 17.0;
    s = s * t2 + 1.0 / 15.0;
    s = s * t2 + 1.0 / 13.0;
    s = s * t2 + 1.0 / 11.0;
    s = s * t2 + 1.0 / 9.0;
    s = s * t2 + 1.0 / 7.0;
    s = s * t2 + 1.0 / 5.0;
    s = s * t2 + 1.0 / 3.0;
    s = s * t2 + 1.0;
    return (double)e * LN2 + 2.0 * t * s;
}

/*
 * cos and sin of 2 pi f for f in [0, 1): quadrant q = floor(4 f) and
 * theta = (4 f - q) pi/2 in [0, pi/2); Taylor series of sin and cos through
 * theta^17 and theta^18 (truncation below 3e-12 relative), then the quadrant
 * rotation.
 */
static inline void cos_sin_turn(double f, double* c, double* s) {
    double x = 4.0 * f;
    int q = (int)x;
    double th = (x - (double)q) * HALF_PI;
    double t2 = th * th;
    /* sin: th (1 - t2/3! + t2^2/5! - ...) */
    double sn = -1.0 / 355687428096000.0; /* -1/17! */
    sn = sn * t2 + 1.0 / 1307674368000.0;  /* 1/15! */
    sn = sn * t2 - 1.0 / 6227020800.0;     /* 1/13! */
    sn = sn * t2 + 1.0 / 39916800.0;       /* 1/11! */
    sn = sn * t2 - 1.0 / 362880.0;         /* 1/9! */
    sn = sn * t2 + 1.0 / 5040.0;           /* 1/7! */
    sn = sn * t2 - 1.0 / 120.0;            /* 1/5! */
    sn = sn * t2 + 1.0 / 6.0;              /* 1/3! */
    sn = th - th * t2 * sn;
    double cs = 1.0 / 6402373705728000.0; /* 1/18! */
    cs = cs * t2 - 1.0 / 20922789888000.0; /* 1/16! */
    cs = cs * t2 + 1.0 / 87178291200.0;    /* 1/14! */
    cs = cs * t2 - 1.0 / 479001600.0;      /* 1/12! */
    cs = cs * t2 + 1.0 / 3628800.0;        /* 1/10! */
    cs = cs * t2 - 1.0 / 40320.0;          /* 1/8! */
    cs = cs * t2 + 1.0 / 720.0;            /* 1/6! */
    cs = cs * t2 - 1.0 / 24.0;             /* 1/4! */
    cs = cs * t2 + 0.5;                    /* 1/2! */
    cs = 1.0 - t2 * cs;
    switch (q & 3) {
        case 0: *c = cs; *s = sn; break;
        case 1: *c = -sn; *s = cs; break;
        case 2: *c = -cs; *s = -sn; break;
        default: *c = sn; *s = -cs; break;
    }
}

static inline void box_muller(uint32_t xe, uint32_t xo, double* n0, double* n1) {
    double u1 = ((double)xe + 0.5) * INV_2_32;
    double u2 = (double)xo * INV_2_32;
    double r2 = -2.0 * ln_unit(u1);
    double r = sqrt(r2); /* IEEE sqrt is correctly rounded */
    double c, s;
    cos_sin_turn(u2, &c, &s);
    *n0 = r * c;
    *n1 = r * s;
}

/* exported for the generator's own accuracy tests */
double synth_ln_unit(double u) { return ln_unit(u); }
void synth_cos_sin_turn(double f, double* c, double* s) { cos_sin_turn(f, c, s); }

/* float -> IEEE binary16, round to nearest even (handles subnormals, inf, nan). */
static inline uint16_t f32_to_f16_rne(float f) {
    uint32_t x;
    memcpy(&x, &f, 4);
    uint32_t sign = (x >> 16) & 0x8000u;
    uint32_t ax = x & 0x7FFFFFFFu;
    if (ax >= 0x7F800000u) { /* inf or nan */
        return (uint16_t)(sign | 0x7C00u | (ax > 0x7F800000u ? 0x200u : 0u));
    }
    if (ax >= 0x477FF000u) { /* rounds to >= 65520 -> inf */
        return (uint16_t)(sign | 0x7C00u);
    }
    if (ax < 0x38800000u) { /* below the smallest normal half: 2^-14 */
        if (ax < 0x33000000u) return (uint16_t)sign; /* < 2^-25 rounds to 0 */
        uint32_t e = ax >> 23;
        uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
        uint32_t shift = 126u - e; /* 14..24: value = m * 2^(e-150), half subnormal unit 2^-24 */
        uint32_t q = m >> shift;
        uint32_t rem = m & ((1u << shift) - 1u);
        uint32_t halfway = 1u << (shift - 1u);
        if (rem > halfway || (rem == halfway && (q & 1u))) q += 1u;
        return (uint16_t)(sign | q);
    }
    uint32_t e = (ax >> 23) - 112u; /* rebias 127 -> 15 */
    uint32_t m = ax & 0x7FFFFFu;
    uint32_t q = (e << 10) | (m >> 13);
    uint32_t rem = m & 0x1FFFu;
    if (rem > 0x1000u || (rem == 0x1000u && (q & 1u))) q += 1u; /* carry may bump exponent: fine */
    return (uint16_t)(sign | q);
}

/* float -> bfloat16, round to nearest even. */
static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t x;
    memcpy(&x, &f, 4);
    if ((x & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((x >> 16) | 0x40u); /* quiet nan */
    uint32_t lsb = (x >> 16) & 1u;
    x += 0x7FFFu + lsb;
    return (uint16_t)(x >> 16);
}

uint16_t synth_f32_to_f16(float f) { return f32_to_f16_rne(f); }
uint16_t synth_f32_to_bf16(float f) { return f32_to_bf16_rne(f); }

enum { SYNTH_F32 = 0, SYNTH_F16 = 1, SYNTH_BF16 = 2 };

/*
 * Fill out[0..n) with draws mean + std * N(0,1) of (seed, stream), elements
 * offset .. offset+n of the stream.  kind selects the storage type.
 */
void synth_normal(uint64_t seed, uint64_t stream, uint64_t offset, uint64_t n, double mean,
                  double std, int kind, void* out) {
    const int64_t CH = 4096; /* elements per parallel chunk, a multiple of 4 */
    int64_t first_chunk = (int64_t)(offset / CH);
    int64_t last_chunk = n ? (int64_t)((offset + n - 1) / CH) : first_chunk - 1;
#pragma omp parallel for schedule(static)
    for (int64_t ch = first_chunk; ch <= last_chunk; ++ch) {
        uint64_t lo = (uint64_t)ch * CH, hi = lo + CH;
        if (lo < offset) lo = offset;
        if (hi > offset + n) hi = offset + n;
        uint64_t i = lo & ~(uint64_t)3;
        for (; i < hi; i += 4) {
            uint32_t x[4];
            philox_block(seed, stream, i >> 2, x);
            double z[4];
            box_muller(x[0], x[1], &z[0], &z[1]);
            box_muller(x[2], x[3], &z[2], &z[3]);
            for (int j = 0; j < 4; ++j) {
                uint64_t e = i + (uint64_t)j;
                if (e < lo || e >= hi) continue;
                float v = (float)(mean + std * z[j]);
                uint64_t o = e - offset;
                if (kind == SYNTH_F32)
                    ((float*)out)[o] = v;
                else if (kind == SYNTH_F16)
                    ((uint16_t*)out)[o] = f32_to_f16_rne(v);
                else
                    ((uint16_t*)out)[o] = f32_to_bf16_rne(v);
            }
        }
    }
}

/* Uniform integers in [lo, hi): lo + floor(x0 * (hi - lo) / 2^32), word x0..x3 of block i/4. */
void synth_uniform_int(uint64_t seed, uint64_t stream, uint64_t n, int32_t lo, int32_t hi,
                       int32_t* out) {
    uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo);
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < (int64_t)((n + 3) / 4); ++b) {
        uint32_t x[4];
        philox_block(seed, stream, (uint64_t)b, x);
        for (int j = 0; j < 4; ++j) {
            uint64_t e = (uint64_t)b * 4 + (uint64_t)j;
            if (e >= n) break;
            out[e] = (int32_t)((int64_t)lo + (int64_t)(((uint64_t)x[j] * span) >> 32));
        }
    }
}

/* Constant fill in a storage type (used for zero LoRA B and similar special cases). */
void synth_const(uint64_t n, double value, int kind, void* out) {
    float v = (float)value;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        if (kind == SYNTH_F32)
            ((float*)out)[i] = v;
        else if (kind == SYNTH_F16)
            ((uint16_t*)out)[i] = f32_to_f16_rne(v);
        else
            ((uint16_t*)out)[i] = f32_to_bf16_rne(v);
    }
}
