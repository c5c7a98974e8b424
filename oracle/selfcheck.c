/*
 * selfcheck.c -- a C driver that runs the oracle's pins without Python, so the
 * oracle can be built and checked under AddressSanitizer and
 * UndefinedBehaviorSanitizer (TEST INFRASTRUCTURE ONLY, like oracle.c).
 *
 *   selfcheck <golden dir>     exit status 0 when every check passes
 *
 * What pins what (each check compares the oracle with something other than
 * itself):
 *   - BF16 cast: the worked examples of tests/golden/bf16_rne_examples.txt
 *     (App. A.2 cell rule, App. D round-to-nearest-even), and the integer
 *     rounding formula (add 0x7FFF plus the kept LSB, then truncate) over a
 *     strided sweep of all 2^32 FP32 patterns plus every pattern next to a
 *     rounding tie; NaNs keep sign and payload and get the quiet bit.
 *   - Encode / apply (Alg. 1): count = number of bitwise mismatches, entries
 *     ascending, apply(snapshot, patch) = cast(w_new) (lossless decode),
 *     capacity truncation, append position, refresh of emitted entries only.
 *   - PULSELoCo sparsify (Alg. 2): a = delta + e; every element either kept
 *     (value a, residual +0) or not (residual a); count = |{|a| >= tau}|;
 *     tau = 0 and tau = +inf.
 *   - Outer step: with no workers the update is the momentum decay; entries
 *     outside the tensor change nothing.
 *   - Delta-varint stream (App. H.2, F.3): tests/golden/varint_examples.txt,
 *     round trips, a stream cut inside a number is rejected.
 *   - 2-D COO downcast (App. H.2 step 4, H.4.1): tests/golden/coo_examples.txt,
 *     round trips, malformed pairs are rejected.
 *   - FP8 E4M3 / MXFP4 receivers (App. D): every FP8 code decodes and
 *     re-encodes to itself, saturation, tests/golden/mxfp4_examples.txt,
 *     encode/apply round trips, the low-precision gate's bookkeeping.
 *   - SHA-256 (App. J.4): the FIPS 180-4 example digests ("abc", the empty
 *     message, the two-block message); the tree of one and of three leaves
 *     written out by hand.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* the oracle's entry points (oracle.c) */
uint16_t oracle_bf16_rne(float x);
void oracle_cast(const float *src, uint16_t *dst, uint64_t n);
uint64_t oracle_encode(const float *w_new, const uint16_t *snap, uint64_t n, uint32_t index_base,
                       uint32_t *idx, uint16_t *val, uint64_t capacity, uint64_t count_in,
                       uint16_t *refresh);
uint64_t oracle_apply(uint16_t *dst, uint64_t n, const uint32_t *idx, const uint16_t *val,
                      uint64_t begin, uint64_t end, uint32_t index_base);
uint64_t oracle_loco(const float *delta, float *residual, uint64_t n, float tau,
                     const float *theta, uint32_t index_base, uint32_t *idx, float *val,
                     uint64_t capacity, uint64_t count_in);
int oracle_outer_step(float *theta, float *momentum, uint64_t n, uint32_t index_base,
                      uint32_t nlists, const uint32_t *const *idx, const float *const *val,
                      const uint64_t *count, float mu, float alpha);
uint64_t oracle_varint_encode(const uint32_t *idx, uint64_t count, uint8_t *out,
                              uint64_t out_capacity);
int64_t oracle_varint_decode(const uint8_t *in, uint64_t nbytes, uint32_t *out, uint64_t max_out);
uint64_t oracle_coo_encode(const uint32_t *idx, uint64_t nent, const uint64_t *seg_begin,
                           uint32_t nseg, const uint32_t *cols, uint32_t *first, uint8_t *drow,
                           uint16_t *dcol, uint64_t out_capacity, uint64_t *seg_pairs);
int64_t oracle_coo_decode(const uint8_t *drow, const uint16_t *dcol, uint64_t npairs,
                          const uint64_t *seg_pairs, const uint64_t *seg_begin, uint32_t nseg,
                          uint64_t nent, const uint32_t *cols, const uint32_t *first,
                          uint32_t *out);
uint8_t oracle_fp8_e4m3(float y);
double oracle_fp8_value(uint8_t c);
void oracle_cast_fp8(const float *x, uint8_t *out, uint64_t n, float inv_scale);
void oracle_cast_mxfp4(const float *x, uint64_t n, uint8_t *codes, uint8_t *scales);
uint64_t oracle_encode_fp8(const float *w_new, const uint8_t *snap, uint64_t n, float inv_scale,
                           uint32_t index_base, uint32_t *idx, uint8_t *val, uint64_t capacity,
                           uint64_t count_in);
uint64_t oracle_encode_mxfp4(const float *w_new, const uint8_t *snap_codes,
                             const uint8_t *snap_scales, uint64_t n, uint32_t index_base,
                             uint32_t *idx, uint16_t *val, uint64_t capacity, uint64_t count_in);
uint64_t oracle_apply_fp8(uint8_t *dst, uint64_t n, const uint32_t *idx, const uint8_t *val,
                          uint64_t begin, uint64_t end, uint32_t index_base);
uint64_t oracle_apply_mxfp4(uint8_t *codes, uint8_t *scales, uint64_t n, const uint32_t *idx,
                            const uint16_t *val, uint64_t begin, uint64_t end, uint32_t index_base);
uint64_t oracle_loco_gate_lp(int dtype, float inv_scale, const float *delta, float *residual,
                             uint64_t n, const float *theta, uint32_t index_base, uint32_t *idx,
                             float *val, uint64_t capacity, uint64_t count_in);
void oracle_sha256(const uint8_t *msg, uint64_t len, uint8_t out[32]);
void oracle_leaf_hashes(const uint8_t *stream, uint64_t nbytes, uint64_t leaf_bytes,
                        uint8_t *digests);
void oracle_merkle_root(const uint8_t *digests, uint64_t nleaves, uint8_t root[32]);

static long n_checks, n_failed;

static void check(int ok, const char *what, long detail)
{
    n_checks++;
    if (!ok) {
        n_failed++;
        if (n_failed <= 20)
            fprintf(stderr, "FAILED: %s (%ld)\n", what, detail);
    }
}

/* xorshift64*: seeded test inputs */
static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t rnd(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1Dull;
}
static double unit(void) { return (double)(rnd() >> 11) * (1.0 / 9007199254740992.0); }
static float gauss(float sd)
{
    double u = unit(), v = unit();
    if (u < 1e-300)
        u = 1e-300;
    return (float)(sd * sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v));
}

static float f_from(uint32_t u)
{
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static void *xmalloc(size_t n)
{
    void *p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "selfcheck: out of memory\n");
        exit(2);
    }
    return p;
}

static FILE *open_golden(const char *dir, const char *name)
{
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE *f = fopen(path, "r");
    if (!f) {
        fprintf(stderr, "selfcheck: cannot open %s\n", path);
        exit(2);
    }
    return f;
}

/* ---------------------------------------------------------------- BF16 cast */

static uint16_t rne_formula(uint32_t u)
{
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)((u >> 16) | 0x40);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

static void check_cast(const char *dir)
{
    FILE *f = open_golden(dir, "bf16_rne_examples.txt");
    char line[512];
    int rows = 0;
    while (fgets(line, sizeof line, f)) {
        unsigned x, b;
        if (line[0] == '#' || sscanf(line, "%x %x", &x, &b) != 2)
            continue;
        check(oracle_bf16_rne(f_from(x)) == (uint16_t)b, "bf16 golden example", (long)x);
        rows++;
    }
    fclose(f);
    check(rows >= 10, "bf16 golden file has its examples", rows);
    for (uint64_t u = 0; u < (1ull << 32); u += 251)
        check(oracle_bf16_rne(f_from((uint32_t)u)) == rne_formula((uint32_t)u), "bf16 sweep",
              (long)u);
    for (uint32_t hi = 0; hi < 0x10000u; hi += 7) /* around each tie of sampled grid points */
        for (int d = -2; d <= 2; d++) {
            uint32_t u = (hi << 16) + 0x8000u + (uint32_t)d;
            check(oracle_bf16_rne(f_from(u)) == rne_formula(u), "bf16 near tie", (long)u);
        }
}

/* ---------------------------------------------------------------- encode / apply */

static void check_codec(void)
{
    static const uint64_t sizes[] = {0, 1, 7, 8, 9, 63, 64, 65, 1000, 4097, 65537};
    for (size_t si = 0; si < sizeof sizes / sizeof sizes[0]; si++) {
        uint64_t n = sizes[si];
        float *w = xmalloc(n * 4), *w2 = xmalloc(n * 4);
        uint16_t *s = xmalloc(n * 2), *r = xmalloc(n * 2), *c = xmalloc(n * 2), *v = xmalloc(n * 2);
        uint32_t *ix = xmalloc(n * 4);
        for (uint64_t i = 0; i < n; i++) {
            w[i] = gauss(0.1414f);
            w2[i] = (rnd() % 16 == 0) ? w[i] + gauss(0.01f) : w[i];
        }
        oracle_cast(w, s, n);
        oracle_cast(w2, c, n);
        uint64_t mism = 0;
        for (uint64_t i = 0; i < n; i++)
            mism += c[i] != s[i];
        memcpy(r, s, n * 2);
        uint64_t cnt = oracle_encode(w2, s, n, 5, ix, v, n, 0, NULL);
        check(cnt == mism, "encode count = mismatches", (long)n);
        for (uint64_t k = 1; k < cnt; k++)
            check(ix[k] > ix[k - 1], "encode indices ascending", (long)k);
        check(oracle_apply(r, n, ix, v, 0, cnt, 5) == 0, "apply rejects nothing", (long)n);
        check(memcmp(r, c, n * 2) == 0, "apply(snapshot, patch) = cast(w_new)", (long)n);
        /* capacity, append position, refresh of emitted entries only */
        uint64_t cap = cnt / 2 + 3;
        memcpy(r, s, n * 2);
        uint64_t cnt2 = oracle_encode(w2, s, n, 5, ix, v, cap, 3, r);
        check(cnt2 == cnt + 3, "append position adds", (long)n);
        uint64_t emitted = cap > 3 ? (cnt < cap - 3 ? cnt : cap - 3) : 0;
        uint64_t changed = 0;
        for (uint64_t i = 0; i < n; i++)
            changed += r[i] != s[i];
        check(changed == emitted, "refresh only emitted entries", (long)n);
        /* out-of-range entries are counted, not written */
        if (n > 0) {
            uint32_t bad[2] = {4, (uint32_t)(5 + n)};
            uint16_t bv[2] = {1, 2};
            check(oracle_apply(r, n, bad, bv, 0, 2, 5) == 2, "apply rejects outside", (long)n);
        }
        free(w), free(w2), free(s), free(r), free(c), free(v), free(ix);
    }
}

/* ---------------------------------------------------------------- PULSELoCo */

static void check_loco(void)
{
    const uint64_t n = 5000;
    float *d = xmalloc(n * 4), *e = xmalloc(n * 4), *e0 = xmalloc(n * 4), *val = xmalloc(n * 4);
    float *th = xmalloc(n * 4);
    uint32_t *ix = xmalloc(n * 4);
    for (uint64_t i = 0; i < n; i++) {
        float g = gauss(1.0f);
        d[i] = gauss(0.00316f) * g * g;
        e0[i] = (rnd() % 3 == 0) ? gauss(0.001f) : 0.0f;
        th[i] = gauss(0.1414f);
    }
    const float taus[] = {0.0f, 0.003f, INFINITY};
    for (int t = 0; t < 3; t++) {
        memcpy(e, e0, n * 4);
        uint64_t cnt = oracle_loco(d, e, n, taus[t], NULL, 0, ix, val, n, 0);
        uint64_t want = 0, k = 0;
        int ok = 1;
        for (uint64_t i = 0; i < n; i++) {
            float a = d[i] + e0[i];
            int keep = fabsf(a) >= taus[t];
            want += keep;
            if (keep) {
                ok &= k < cnt && ix[k] == i && val[k] == a && e[i] == 0.0f && !signbit(e[i]);
                k++;
            } else {
                ok &= e[i] == a;
            }
        }
        check(cnt == want, "loco count = |{|a| >= tau}|", t);
        check(ok, "loco partition and residual", t);
    }
    /* BF16 gate and the low-precision gates: kept <=> residual +0 and value a */
    for (int dtype = 0; dtype <= 2; dtype++) {
        memcpy(e, e0, n * 4);
        uint64_t cnt = dtype == 0 ? oracle_loco(d, e, n, 0.0f, th, 0, ix, val, n, 0)
                                  : oracle_loco_gate_lp(dtype, 64.0f, d, e, n, th, 0, ix, val, n, 0);
        uint64_t k = 0;
        int ok = 1;
        for (uint64_t i = 0; i < n; i++) {
            float a = d[i] + e0[i];
            if (k < cnt && ix[k] == i) {
                ok &= val[k] == a && e[i] == 0.0f;
                k++;
            } else {
                ok &= e[i] == a;
            }
        }
        check(ok && k == cnt, "gate bookkeeping", dtype);
    }
    free(d), free(e), free(e0), free(val), free(th), free(ix);
}

static void check_outer(void)
{
    const uint64_t n = 300;
    float th[300], m[300], th2[300], m2[300];
    for (uint64_t i = 0; i < n; i++) {
        th[i] = th2[i] = gauss(0.1f);
        m[i] = m2[i] = gauss(0.01f);
    }
    check(oracle_outer_step(th, m, n, 0, 0, NULL, NULL, NULL, 0.5f, 0.25f) == 0, "outer rc", 0);
    int ok = 1;
    for (uint64_t i = 0; i < n; i++) {
        float mm = 0.5f * m2[i]; /* no workers: g = 0, m <- mu m, theta <- theta - alpha mu m */
        float t = 0.5f * mm;
        ok &= m[i] == mm && th[i] == th2[i] - 0.25f * t;
    }
    check(ok, "outer step without workers decays the momentum", 0);
    /* entries outside [base, base + n) change nothing */
    uint32_t ia[3] = {3, 50, 60}, ib[5] = {1, 3, 50, 60, 400};
    float va[3] = {1.0f, 2.0f, 3.0f}, vb[5] = {9.0f, 1.0f, 2.0f, 3.0f, 9.0f};
    const uint32_t *pa[1] = {ia}, *pb[1] = {ib};
    const float *qa[1] = {va}, *qb[1] = {vb};
    uint64_t ca[1] = {3}, cb[1] = {5};
    memcpy(th2, th, sizeof th);
    memcpy(m2, m, sizeof m);
    oracle_outer_step(th, m, n, 2, 1, pa, qa, ca, 0.9f, 0.7f);
    oracle_outer_step(th2, m2, n, 2, 1, pb, qb, cb, 0.9f, 0.7f);
    check(memcmp(th, th2, sizeof th) == 0 && memcmp(m, m2, sizeof m) == 0,
          "outer step ignores indices outside the tensor", 0);
}

/* ---------------------------------------------------------------- index streams */

static void check_varint(const char *dir)
{
    FILE *f = open_golden(dir, "varint_examples.txt");
    char line[512];
    int rows = 0;
    while (fgets(line, sizeof line, f)) {
        unsigned long num;
        int used = 0;
        if (line[0] == '#' || sscanf(line, "%lu%n", &num, &used) != 1)
            continue;
        uint8_t want[8], got[8];
        int nb = 0;
        unsigned byte;
        const char *p = line + used;
        int adv;
        while (nb < 8 && sscanf(p, "%x%n", &byte, &adv) == 1) {
            want[nb++] = (uint8_t)byte;
            p += adv;
        }
        uint32_t one = (uint32_t)num;
        uint64_t len = oracle_varint_encode(&one, 1, got, sizeof got);
        check(len == (uint64_t)nb && memcmp(got, want, (size_t)nb) == 0, "varint golden", (long)num);
        rows++;
    }
    fclose(f);
    check(rows >= 10, "varint golden file has its examples", rows);
    const uint64_t n = 20000;
    uint32_t *ix = xmalloc(n * 4), *back = xmalloc(n * 4);
    uint8_t *buf = xmalloc(n * 5);
    uint32_t x = 0;
    for (uint64_t k = 0; k < n; k++) {
        x += 1 + (uint32_t)(rnd() % (k % 97 == 0 ? 3000000u : 300u));
        ix[k] = x;
    }
    uint64_t len = oracle_varint_encode(ix, n, buf, n * 5);
    check(oracle_varint_decode(buf, len, back, n) == (int64_t)n, "varint decode count", 0);
    check(memcmp(ix, back, n * 4) == 0, "varint round trip", 0);
    buf[len - 1] |= 0x80; /* the last number no longer ends */
    check(oracle_varint_decode(buf, len, back, n) == -1, "varint cut stream rejected", 0);
    free(ix), free(back), free(buf);
}

static void check_coo(const char *dir)
{
    FILE *f = open_golden(dir, "coo_examples.txt");
    char line[1024];
    int rows = 0;
    while (fgets(line, sizeof line, f)) {
        if (line[0] == '#')
            continue;
        char *bar1 = strchr(line, '|');
        if (!bar1)
            continue;
        char *bar2 = strchr(bar1 + 1, '|'), *bar3 = bar2 ? strchr(bar2 + 1, '|') : NULL;
        if (!bar3)
            continue;
        uint32_t cols = (uint32_t)strtoul(line, NULL, 10);
        uint32_t ix[64], first_want = (uint32_t)strtoul(bar2 + 1, NULL, 10);
        uint64_t ne = 0;
        for (char *p = bar1 + 1; p < bar2 && ne < 64;) {
            char *end;
            unsigned long v = strtoul(p, &end, 10);
            if (end == p)
                break;
            ix[ne++] = (uint32_t)v;
            p = end;
        }
        uint8_t wr[64], dr[64];
        uint16_t wc[64], dc[64];
        uint64_t np_want = 0;
        for (char *p = bar3 + 1; np_want < 64;) {
            char *end;
            unsigned long a = strtoul(p, &end, 10);
            if (end == p || *end != ':')
                break;
            unsigned long b = strtoul(end + 1, &end, 10);
            wr[np_want] = (uint8_t)a;
            wc[np_want] = (uint16_t)b;
            np_want++;
            p = end;
        }
        uint64_t sb[1] = {0}, sp[1];
        uint32_t first[1], back[64];
        uint64_t np = oracle_coo_encode(ix, ne, sb, 1, &cols, first, dr, dc, 64, sp);
        int ok = np == np_want && first[0] == first_want;
        for (uint64_t q = 0; ok && q < np; q++)
            ok = dr[q] == wr[q] && dc[q] == wc[q];
        check(ok, "coo golden", rows);
        check(oracle_coo_decode(dr, dc, np, sp, sb, 1, ne, &cols, first, back) == (int64_t)ne &&
                  memcmp(back, ix, ne * 4) == 0,
              "coo golden decodes", rows);
        rows++;
    }
    fclose(f);
    check(rows >= 5, "coo golden file has its examples", rows);
    /* random round trip over three segments */
    const uint64_t ne = 6000;
    uint32_t *ix = xmalloc(ne * 4), *back = xmalloc(ne * 4), first[3];
    uint64_t sb[3] = {0, 1000, 4000}, sp[3];
    uint32_t cols[3] = {7, 5120, 65535};
    for (int s = 0; s < 3; s++) {
        uint64_t e = s < 2 ? sb[s + 1] : ne;
        uint32_t x = (uint32_t)(rnd() % 50);
        for (uint64_t k = sb[s]; k < e; k++) {
            ix[k] = x;
            x += 1 + (uint32_t)(rnd() % (k % 50 == 0 ? 4000000u : 900u));
        }
    }
    /* a first pass with no room counts the pairs (escapes included) */
    uint64_t np = oracle_coo_encode(ix, ne, sb, 3, cols, first, NULL, NULL, 0, sp);
    uint8_t *dr = xmalloc(np);
    uint16_t *dc = xmalloc(np * 2);
    check(oracle_coo_encode(ix, ne, sb, 3, cols, first, dr, dc, np, sp) == np, "coo pairs", 0);
    check(oracle_coo_decode(dr, dc, np, sp, sb, 3, ne, cols, first, back) == (int64_t)ne &&
              memcmp(back, ix, ne * 4) == 0,
          "coo round trip", 0);
    uint8_t d0 = dr[5];
    uint16_t c0 = dc[5];
    dr[5] = 0, dc[5] = 0; /* a same-row pair with no column step: no encoder writes it */
    check(oracle_coo_decode(dr, dc, np, sp, sb, 3, ne, cols, first, back) == -1,
          "coo malformed pair rejected", 0);
    dr[5] = d0, dc[5] = c0;
    free(ix), free(back), free(dr), free(dc);
}

/* ---------------------------------------------------------------- FP8 / MXFP4 */

static void check_lowp(const char *dir)
{
    for (int c = 0; c < 256; c++) {
        if ((c & 0x7F) == 0x7F)
            continue;
        check(oracle_fp8_e4m3((float)oracle_fp8_value((uint8_t)c)) == c, "fp8 code round trip", c);
    }
    check(oracle_fp8_e4m3(1e6f) == 0x7E && oracle_fp8_e4m3(-INFINITY) == 0xFE, "fp8 saturates", 0);
    check((oracle_fp8_e4m3(NAN) & 0x7F) == 0x7F, "fp8 NaN", 0);

    FILE *f = open_golden(dir, "mxfp4_examples.txt");
    char line[512];
    int rows = 0;
    while (fgets(line, sizeof line, f)) {
        if (line[0] == '#')
            continue;
        char *bar1 = strchr(line, '|');
        if (!bar1)
            continue;
        char *bar2 = strchr(bar1 + 1, '|');
        if (!bar2)
            continue;
        float x[32];
        uint64_t nx = 0;
        for (char *p = line; p < bar1 && nx < 32;) {
            char *end;
            double v = strtod(p, &end);
            if (end == p)
                break;
            x[nx++] = (float)v;
            p = end;
            while (*p == ',' || *p == ' ')
                p++;
        }
        unsigned scale = (unsigned)strtoul(bar1 + 1, NULL, 10);
        uint8_t codes[16], sc[1];
        oracle_cast_mxfp4(x, nx, codes, sc);
        int ok = sc[0] == scale;
        char *p = bar2 + 1;
        for (uint64_t i = 0; i < nx; i++) {
            char *end;
            unsigned long want = strtoul(p, &end, 16);
            ok &= end != p && ((codes[i / 2] >> (4 * (i & 1))) & 0xF) == want;
            p = end;
        }
        check(ok, "mxfp4 golden block", rows);
        rows++;
    }
    fclose(f);
    check(rows == 12, "mxfp4 golden file has its examples", rows);

    /* encode/apply round trips: the receiver copy equals cast_D(w_new) afterwards */
    const uint64_t n = 3000;
    float *w = xmalloc(n * 4), *w2 = xmalloc(n * 4);
    uint8_t *f0 = xmalloc(n), *f1 = xmalloc(n), *fv = xmalloc(n);
    uint8_t *c0 = xmalloc(n), *s0 = xmalloc(n), *c1 = xmalloc(n), *s1 = xmalloc(n);
    uint16_t *mv = xmalloc(n * 2);
    uint32_t *ix = xmalloc(n * 4);
    for (uint64_t i = 0; i < n; i++) {
        w[i] = gauss(0.1414f);
        w2[i] = (rnd() % 8 == 0) ? w[i] * 1.5f : w[i];
    }
    oracle_cast_fp8(w, f0, n, 40.0f);
    oracle_cast_fp8(w2, f1, n, 40.0f);
    uint64_t cnt = oracle_encode_fp8(w2, f0, n, 40.0f, 0, ix, fv, n, 0);
    check(oracle_apply_fp8(f0, n, ix, fv, 0, cnt, 0) == 0 && memcmp(f0, f1, n) == 0,
          "fp8 encode/apply round trip", (long)cnt);
    oracle_cast_mxfp4(w, n, c0, s0);
    oracle_cast_mxfp4(w2, n, c1, s1);
    cnt = oracle_encode_mxfp4(w2, c0, s0, n, 0, ix, mv, n, 0);
    check(oracle_apply_mxfp4(c0, s0, n, ix, mv, 0, cnt, 0) == 0 &&
              memcmp(c0, c1, (n + 1) / 2) == 0 && memcmp(s0, s1, (n + 31) / 32) == 0,
          "mxfp4 encode/apply round trip", (long)cnt);
    free(w), free(w2), free(f0), free(f1), free(fv), free(c0), free(s0), free(c1), free(s1);
    free(mv), free(ix);
}

/* ---------------------------------------------------------------- SHA-256 */

static int hex_eq(const uint8_t d[32], const char *hex)
{
    for (int i = 0; i < 32; i++) {
        unsigned b;
        if (sscanf(hex + 2 * i, "%2x", &b) != 1 || d[i] != b)
            return 0;
    }
    return 1;
}

static void check_hash(void)
{
    uint8_t d[32];
    oracle_sha256((const uint8_t *)"abc", 3, d);
    check(hex_eq(d, "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"),
          "sha256 abc", 0);
    oracle_sha256(NULL, 0, d);
    check(hex_eq(d, "e3b0c44298fc1c149afbf4c8996fb92427ae41e4649b934ca495991b7852b855"),
          "sha256 empty", 0);
    const char *m2 = "abcdbcdecdefdefgefghfghighijhijkijkljklmklmnlmnomnopnopq";
    oracle_sha256((const uint8_t *)m2, strlen(m2), d);
    check(hex_eq(d, "248d6a61d20638b8e5c026930c3e6039a33ce45964ff2167f6ecedd419db06c1"),
          "sha256 two blocks", 0);
    /* tree by hand: one leaf is its leaf hash; three leaves are
     * node(node(l0, l1), l2), node(a, b) = SHA-256(0x01 || a || b),
     * leaf(c) = SHA-256(0x00 || c) */
    uint8_t stream[100], leaves[3 * 32], root[32], buf[65], n01[32], want[32];
    for (int i = 0; i < 100; i++)
        stream[i] = (uint8_t)(rnd() & 0xFF);
    oracle_leaf_hashes(stream, 100, 40, leaves);
    buf[0] = 0x00;
    memcpy(buf + 1, stream, 40);
    oracle_sha256(buf, 41, d);
    check(memcmp(d, leaves, 32) == 0, "leaf hash = SHA-256(0x00 || chunk)", 0);
    oracle_merkle_root(leaves, 1, root);
    check(memcmp(root, leaves, 32) == 0, "one leaf is the root", 0);
    oracle_merkle_root(leaves, 3, root);
    buf[0] = 0x01;
    memcpy(buf + 1, leaves, 64);
    oracle_sha256(buf, 65, n01);
    memcpy(buf + 1, n01, 32);
    memcpy(buf + 33, leaves + 64, 32);
    oracle_sha256(buf, 65, want);
    check(memcmp(root, want, 32) == 0, "three-leaf tree", 0);
}

int main(int argc, char **argv)
{
    if (argc != 2) {
        fprintf(stderr, "usage: %s <golden dir>\n", argv[0]);
        return 2;
    }
    check_cast(argv[1]);
    check_codec();
    check_loco();
    check_outer();
    check_varint(argv[1]);
    check_coo(argv[1]);
    check_lowp(argv[1]);
    check_hash();
    if (n_failed) {
        fprintf(stderr, "selfcheck: %ld of %ld checks failed\n", n_failed, n_checks);
        return 1;
    }
    printf("selfcheck: %ld checks passed\n", n_checks);
    return 0;
}
