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

/*
 * float -> IEEE binary16, round to nearest even (subnormals, inf and nan
 * included).  Every case is computed and the right one selected, so the
 * conversion loop runs as vector code:
 *   normal half (|x| >= 2^-14): exponent rebiased 127 -> 15, mantissa cut
 *   to 10 bits, rounded on the 13 dropped bits (a carry may bump the
 *   exponent, up to inf);
 *   subnormal half (2^-25 <= |x| < 2^-14): the 24-bit significand shifted
 *   right by 126 - e (14..24) in units of 2^-24, rounded on the dropped bits;
 *   below 2^-25: zero; rounding to >= 65520: inf; nan stays a quiet nan.
 */
/* 0/1 comparisons and a select on 32-bit values below 2^31, in plain
   arithmetic (no branches, no boolean vectors) */
static inline uint32_t gt31(uint32_t a, uint32_t b) { return (b - a) >> 31; }
static inline uint32_t eq31(uint32_t a, uint32_t b) { return ((a ^ b) - 1u) >> 31; }
static inline uint32_t sel31(uint32_t c, uint32_t a, uint32_t b) {
    uint32_t mask = 0u - c;
    return (a & mask) | (b & ~mask);
}

static inline uint32_t f32_to_f16_bits32(float f) {
    uint32_t x;
    memcpy(&x, &f, 4);
    uint32_t sign = (x >> 16) & 0x8000u;
    uint32_t ax = x & 0x7FFFFFFFu;
    uint32_t e = ax >> 23;
    uint32_t m = ax & 0x7FFFFFu;
    uint32_t qn = ((e - 112u) << 10) | (m >> 13);
    uint32_t remn = m & 0x1FFFu;
    qn += gt31(remn, 0x1000u) | (eq31(remn, 0x1000u) & qn & 1u);
    /* subnormal shift 126 - e, used only for e in [102, 112]; e is clamped
       there so that every shift is defined */
    uint32_t ec = e < 102u ? 102u : e;
    ec = ec > 112u ? 112u : ec;
    uint32_t sh = 126u - ec;
    uint32_t ms = m | 0x800000u;
    uint32_t qs = ms >> sh;
    uint32_t rems = ms & ((1u << sh) - 1u);
    uint32_t half = 1u << (sh - 1u);
    qs += gt31(rems, half) | (eq31(rems, half) & qs & 1u);
    uint32_t r = qn;
    r = sel31(gt31(0x38800000u, ax), qs, r);
    r = sel31(gt31(0x33000000u, ax), 0u, r);
    r = sel31(1u - gt31(0x477FF000u, ax), 0x7C00u, r);
    r = sel31(1u - gt31(0x7F800000u, ax), 0x7C00u | (gt31(ax, 0x7F800000u) << 9), r);
    return sign | r;
}

static inline uint16_t f32_to_f16_rne(float f) { return (uint16_t)f32_to_f16_bits32(f); }

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
 * Draws of NB consecutive Philox blocks (4 NB elements), computed stage by
 * stage over arrays: Philox for every block, then ln and sqrt of every pair,
 * then cos and sin, then the products.  Each stage is a loop without
 * branches that the compiler turns into vector code, and every element goes
 * through exactly the operations of philox_block, ln_unit and cos_sin_turn
 * above, in the same order (selects replace their branches; the exponent is
 * turned into a double by the exact 2^52 trick instead of an integer
 * conversion), so the draws are bit for bit those of the scalar functions.
 */
#define NB 256

static inline uint64_t dbits(double x) {
    uint64_t b;
    memcpy(&b, &x, 8);
    return b;
}

static inline double bdbl(uint64_t b) {
    double x;
    memcpy(&x, &b, 8);
    return x;
}

/* an integer 0 <= k < 2^52 as a double, exactly (2^52 + k has k in its mantissa) */
static inline double small_int(uint64_t k) {
    return bdbl(k | 0x4330000000000000ull) - 4503599627370496.0;
}

/* Box-Muller radius, cos and sin for NB word pairs (x_even, x_odd). */
static inline void pair_stage(const uint32_t* restrict we, const uint32_t* restrict wo,
                              double* restrict rad, double* restrict cs, double* restrict sn) {
    for (int b = 0; b < NB; ++b) {
        /* r = sqrt(-2 ln u1), ln as in ln_unit */
        double u = (small_int(we[b]) + 0.5) * INV_2_32;
        uint64_t bits = dbits(u);
        /* m in [1, 2) from the mantissa; m > sqrt(2) compared on the bit
           patterns (monotone for positive doubles); halving m lowers its
           exponent field by one */
        uint64_t mb = (bits & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull;
        uint64_t big = (uint64_t)((int64_t)mb > (int64_t)0x3FF6A09E667F3BCDull);
        double m = bdbl(mb - (big << 52));
        double ed = small_int(((bits >> 52) & 0x7FFull)) - 1023.0;
        ed = ed + small_int(big);
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
        double ln = ed * LN2 + 2.0 * t * s;
        rad[b] = sqrt(-2.0 * ln);
        /* cos and sin of 2 pi u2, as in cos_sin_turn; the quadrant is the
           integer part of 4 u2 */
        double f = small_int(wo[b]) * INV_2_32;
        double x = 4.0 * f;
        int32_t qi = (int32_t)x;
        double qd = (double)qi;
        double th = (x - qd) * HALF_PI;
        double th2 = th * th;
        double a = -1.0 / 355687428096000.0;
        a = a * th2 + 1.0 / 1307674368000.0;
        a = a * th2 - 1.0 / 6227020800.0;
        a = a * th2 + 1.0 / 39916800.0;
        a = a * th2 - 1.0 / 362880.0;
        a = a * th2 + 1.0 / 5040.0;
        a = a * th2 - 1.0 / 120.0;
        a = a * th2 + 1.0 / 6.0;
        a = th - th * th2 * a;
        double c = 1.0 / 6402373705728000.0;
        c = c * th2 - 1.0 / 20922789888000.0;
        c = c * th2 + 1.0 / 87178291200.0;
        c = c * th2 - 1.0 / 479001600.0;
        c = c * th2 + 1.0 / 3628800.0;
        c = c * th2 - 1.0 / 40320.0;
        c = c * th2 + 1.0 / 720.0;
        c = c * th2 - 1.0 / 24.0;
        c = c * th2 + 0.5;
        c = 1.0 - th2 * c;
        /* quadrants 0..3: (cos, sin) = (c, a), (-a, c), (-c, -a), (a, -c):
           swap on odd quadrants, then sign flips, all on the bit patterns */
        uint64_t q = (uint64_t)(int64_t)qi & 3u;
        uint64_t swap = 0 - (q & 1u);
        uint64_t ab = dbits(a), cb = dbits(c);
        uint64_t cvb = (ab & swap) | (cb & ~swap);
        uint64_t svb = (cb & swap) | (ab & ~swap);
        cs[b] = bdbl(cvb ^ (((q ^ (q >> 1)) & 1u) << 63));
        sn[b] = bdbl(svb ^ ((q >> 1) << 63));
    }
}

static void draw_blocks(uint64_t seed, uint64_t stream, uint64_t block0, double z[4 * NB]) {
    uint32_t w0[NB], w1[NB], w2[NB], w3[NB];
    const uint32_t s0 = (uint32_t)stream, s1 = (uint32_t)(stream >> 32);
    for (int b = 0; b < NB; ++b) {
        uint64_t blk = block0 + (uint64_t)b;
        uint32_t c0 = (uint32_t)blk, c1 = (uint32_t)(blk >> 32), c2 = s0, c3 = s1;
        uint32_t ka = (uint32_t)seed, kb = (uint32_t)(seed >> 32);
        for (int r = 0; r < 10; ++r) {
            uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
            uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
            uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ ka;
            uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ kb;
            c0 = n0;
            c1 = (uint32_t)p1;
            c2 = n2;
            c3 = (uint32_t)p0;
            ka += PHILOX_W0;
            kb += PHILOX_W1;
        }
        w0[b] = c0;
        w1[b] = c1;
        w2[b] = c2;
        w3[b] = c3;
    }
    double rad0[NB], cs0[NB], sn0[NB], rad1[NB], cs1[NB], sn1[NB];
    pair_stage(w0, w1, rad0, cs0, sn0); /* words (x0, x1) of each block */
    pair_stage(w2, w3, rad1, cs1, sn1); /* words (x2, x3) */
    for (int b = 0; b < NB; ++b) {
        z[4 * b + 0] = rad0[b] * cs0[b];
        z[4 * b + 1] = rad0[b] * sn0[b];
        z[4 * b + 2] = rad1[b] * cs1[b];
        z[4 * b + 3] = rad1[b] * sn1[b];
    }
}

/*
 * Fill out[0..n) with draws mean + std * N(0,1) of (seed, stream), elements
 * offset .. offset+n of the stream.  kind selects the storage type.
 */
void synth_normal(uint64_t seed, uint64_t stream, uint64_t offset, uint64_t n, double mean,
                  double std, int kind, void* out) {
    const int64_t CH = 4 * NB; /* elements per parallel chunk */
    int64_t first_chunk = (int64_t)(offset / CH);
    int64_t last_chunk = n ? (int64_t)((offset + n - 1) / CH) : first_chunk - 1;
#pragma omp parallel for schedule(static)
    for (int64_t ch = first_chunk; ch <= last_chunk; ++ch) {
        double z[4 * NB];
        uint64_t base = (uint64_t)ch * CH;
        draw_blocks(seed, stream, base >> 2, z);
        uint64_t lo = base < offset ? offset - base : 0;
        uint64_t hi = base + CH > offset + n ? offset + n - base : CH;
        uint64_t o = base + lo - offset;
        float v[4 * NB];
        for (uint64_t j = lo; j < hi; ++j) v[j] = (float)(mean + std * z[j]);
        if (kind == SYNTH_F32) {
            memcpy((float*)out + o, v + lo, (hi - lo) * sizeof(float));
        } else if (kind == SYNTH_F16) {
            uint32_t h[4 * NB]; /* 32-bit lanes for the conversion, narrowed after */
            for (uint64_t j = lo; j < hi; ++j) h[j] = f32_to_f16_bits32(v[j]);
            uint16_t* dst = (uint16_t*)out + o;
            for (uint64_t j = lo; j < hi; ++j) dst[j - lo] = (uint16_t)h[j];
        } else {
            uint16_t* dst = (uint16_t*)out + o;
            for (uint64_t j = lo; j < hi; ++j) dst[j - lo] = f32_to_bf16_rne(v[j]);
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
