/*
 * oracle.c -- plain, single-threaded CPU oracle for the PULSE patch codec.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference the GPU library is
 * checked against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it.  It shares no code, header, table or constant
 * generator with the GPU library and must never be linked into it.
 *
 * Every function below follows a passage of the paper (arXiv 2602.03839,
 * "PULSE: compute-visible sparsification") and is written as the plain
 * definition of what that passage computes, not as a fast kernel:
 *
 *   oracle_bf16_rne      App. A.2, Def. "Update Absorption" (RNE cell rule) and
 *                        App. D (round-to-nearest-even is the rounding mode).
 *   oracle_cast          Sec. 3 "Sparsity metric": the BF16 view of the FP32 master.
 *   oracle_encode        Sec. 4.2, Alg. 1 Encode (changed set and its values) and
 *                        App. H.5, Alg. 3 (per-tensor mask, bitwise compare).
 *   oracle_apply         Sec. 4.2, Alg. 1 Decode (W_t[I] <- V) and App. H.5,
 *                        Alg. 4 (direct value assignment, no FP arithmetic).
 *   oracle_loco          Sec. 4.3, Alg. 2: s = Delta + e, the selection, and the
 *                        error-feedback update e[I] <- 0, e[not I] <- s.
 *   oracle_outer_step    Sec. 4.3, Alg. 2: SparseSync's union-average of the
 *                        workers' selected values, then the outer Nesterov step
 *                        m <- mu m + g, theta <- theta - alpha (mu m + g).
 *   oracle_varint_encode App. H.2 (index encoding: sorted, first index as-is,
 *   oracle_varint_decode then differences) and App. F.3 (PULSELoCo's sparse
 *                        stream: delta-encoded, varint-packed indices).
 *   oracle_coo_encode    App. H.2 step 4 / App. H.4.1 (type downscaling): the
 *   oracle_coo_decode    2-D COO delta stream, uint8 row and uint16 column fields.
 *   oracle_fp8_e4m3,     App. D (lower-precision receivers): the compute view
 *   oracle_cast_fp8,     cast_D for D = FP8 E4M3 and MXFP4, Alg. 1's encode and
 *   oracle_cast_mxfp4,   apply on D-values, and the gate G_D of Alg. 2 for a
 *   oracle_encode_fp8/_mxfp4, oracle_apply_fp8/_mxfp4, oracle_loco_gate_lp
 *                        receiver that computes in D.
 *   oracle_sha256        App. J.4 (weight-level integrity hash): SHA-256 as
 *   oracle_leaf_hashes   FIPS 180-4 defines it, applied as a tree (RFC 6962
 *   oracle_merkle_root   Merkle Tree Hash) over fixed-size chunks of the
 *                        concatenated BF16 bytes.
 *
 * Readings where the paper is silent:
 *   - A NaN input casts to a quiet NaN that keeps the sign and the leading
 *     payload bits (IEEE 754-2019 6.2.3 NaN propagation; the paper never meets NaN).
 *   - Overflow rounds to +-inf exactly as IEEE RNE with an unbounded exponent.
 *   - Subnormals are rounded like any other value (no flush to zero).
 *   - Equality of BF16 values is bitwise, so +0 and -0 differ (Sec. 3 metric).
 *   - The weight hash is a tree of SHA-256 over 16 KiB chunks of the BF16 byte
 *     stream (low byte of each value first), not one SHA-256 over the stream.
 *   - Output entries beyond `capacity` are not written; the returned count is
 *     still the true total.  `refresh` is written only for emitted entries.  In
 *     the sparsifier an entry that was selected but not emitted stays in the
 *     residual (it was not sent, so error feedback keeps it).
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -shared -fPIC -o liboracle.so oracle.c -lm
 * (no FMA contraction is possible: the only FP arithmetic is one add or one
 * subtract per element, and exact double-precision distance comparisons).
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* Scratch allocation that cannot fail silently: the oracle is a checker, so a
 * missing buffer stops the process with a message instead of producing a
 * result. */
static void *oracle_alloc(size_t bytes, int zero)
{
    void *p = zero ? calloc(bytes ? bytes : 1, 1) : malloc(bytes ? bytes : 1);
    if (!p) {
        fprintf(stderr, "oracle: cannot allocate %zu bytes\n", bytes);
        abort();
    }
    return p;
}

static float float_from_bits(uint32_t u)
{
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static uint32_t bits_from_float(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return u;
}

/* Value of a BF16 bit pattern, as a double (every BF16 value is exact in double). */
double oracle_bf16_value(uint16_t b)
{
    return (double)float_from_bits((uint32_t)b << 16);
}

/*
 * FP32 -> BF16, round to nearest, ties to even (App. A.2 and App. D).
 *
 * By definition: take the two BF16 values that bracket x in magnitude -- the
 * truncation `lo` (upper 16 bits of x) and the next BF16 magnitude `hi` --
 * measure both distances exactly in double, return the nearer one, and on a
 * tie return the one whose last mantissa bit is 0.  When `lo` is the largest
 * finite BF16, `hi` is infinity and its distance is measured to 2^128, the
 * value the next step would have with an unbounded exponent (IEEE overflow
 * rule for round-to-nearest).
 */
uint16_t oracle_bf16_rne(float x)
{
    uint32_t u = bits_from_float(x);
    if (isnan(x))
        return (uint16_t)((u >> 16) | 0x0040); /* keep sign and top payload, set the quiet bit */
    uint16_t lo = (uint16_t)(u >> 16);
    if (isinf(x))
        return lo;
    uint16_t hi = (uint16_t)(lo + 1); /* next magnitude, same sign */

    double ax = fabs((double)x);
    double alo = fabs(oracle_bf16_value(lo));
    double ahi = ((hi & 0x7FFF) == 0x7F80) ? ldexp(1.0, 128) : fabs(oracle_bf16_value(hi));
    double d_lo = ax - alo; /* both differences are exact in double */
    double d_hi = ahi - ax;

    if (d_lo < d_hi)
        return lo;
    if (d_hi < d_lo)
        return hi;
    return (lo & 1) ? hi : lo;
}

/* Dense BF16 view of an FP32 tensor: dst[i] = bf16(src[i]). */
void oracle_cast(const float *src, uint16_t *dst, uint64_t n)
{
    for (uint64_t i = 0; i < n; i++)
        dst[i] = oracle_bf16_rne(src[i]);
}

/*
 * Encode one tensor (Alg. 1 Encode, Alg. 3 per-tensor body):
 *   I = { i : bf16(w_new[i]) != snap[i] }   (bitwise),   V = bf16(w_new)[I],
 * emitted in ascending i as (index_base + i, value) at positions
 * count_in, count_in + 1, ...  Returns count_in + |I|.
 */
uint64_t oracle_encode(const float *w_new, const uint16_t *snap, uint64_t n, uint32_t index_base,
                       uint32_t *idx, uint16_t *val, uint64_t capacity, uint64_t count_in,
                       uint16_t *refresh)
{
    uint64_t count = count_in;
    for (uint64_t i = 0; i < n; i++) {
        uint16_t b = oracle_bf16_rne(w_new[i]);
        if (b != snap[i]) {
            if (count < capacity) {
                idx[count] = (uint32_t)(index_base + i);
                val[count] = b;
                if (refresh)
                    refresh[i] = b;
            }
            count++;
        }
    }
    return count;
}

/*
 * Apply a patch (Alg. 1 Decode, Alg. 4): dst[idx[k] - index_base] = val[k]
 * for k in [begin, end).  Entries whose index falls outside the tensor are
 * skipped and counted; the function returns that count.
 */
uint64_t oracle_apply(uint16_t *dst, uint64_t n, const uint32_t *idx, const uint16_t *val,
                      uint64_t begin, uint64_t end, uint32_t index_base)
{
    uint64_t rejected = 0;
    for (uint64_t k = begin; k < end; k++) {
        if (idx[k] < index_base || (uint64_t)(idx[k] - index_base) >= n) {
            rejected++;
            continue;
        }
        dst[idx[k] - index_base] = val[k];
    }
    return rejected;
}

/*
 * PULSELoCo-style sparsification with error feedback (Alg. 2, lines forming
 * s, the selected set, and the residual update):
 *   a_i = fl32(delta_i + e_i)
 *   selected iff |a_i| >= tau                                  (theta == NULL)
 *   selected iff bf16(theta_i) != bf16(fl32(theta_i - a_i))    (theta != NULL,
 *                                          the compute-visibility gate, Sec. 4.1)
 *   selected and emitted:  (index_base + i, a_i) is written, e_i = +0
 *   otherwise:             e_i = a_i
 * Returns count_in + number selected.
 */
uint64_t oracle_loco(const float *delta, float *residual, uint64_t n, float tau,
                     const float *theta, uint32_t index_base, uint32_t *idx, float *val,
                     uint64_t capacity, uint64_t count_in)
{
    uint64_t count = count_in;
    for (uint64_t i = 0; i < n; i++) {
        float a = delta[i] + residual[i];
        int selected;
        if (theta) {
            float after = theta[i] - a;
            selected = oracle_bf16_rne(theta[i]) != oracle_bf16_rne(after);
        } else {
            selected = fabsf(a) >= tau;
        }
        if (selected && count < capacity) {
            idx[count] = (uint32_t)(index_base + i);
            val[count] = a;
            residual[i] = 0.0f;
        } else {
            residual[i] = a;
        }
        if (selected)
            count++;
    }
    return count;
}

/*
 * PULSELoCo outer step (Sec. 4.3, Alg. 2: the SparseSync line and the two
 * outer-optimizer lines after it).
 *
 * SparseSync returns the union of the R workers' selected sets, each value the
 * average over all R workers of what they sent, a worker that did not send an
 * index counting as zero:
 *   g_i = (v_0[i] + v_1[i] + ... + v_{R-1}[i]) / R,  summed left to right in
 *         worker order, starting from +0, with v_r[i] = 0 where worker r sent
 *         nothing; g_i = +0 when R == 0.
 * Then the outer Sutskever-form Nesterov step with momentum mu, step alpha:
 *   m_i     <- mu * m_i + g_i
 *   theta_i <- theta_i - alpha * (mu * m_i + g_i)      (m_i the new momentum)
 * Each operation is rounded to FP32 on its own (no fused multiply-add).
 *
 * Worker r's list is entries [0, count[r]) of idx[r] / val[r], indices of the
 * form index_base + i; an index outside [index_base, index_base + n) is
 * ignored.  Indices within one list are distinct.  Returns 0.
 */
int oracle_outer_step(float *theta, float *momentum, uint64_t n, uint32_t index_base,
                      uint32_t nlists, const uint32_t *const *idx, const float *const *val,
                      const uint64_t *count, float mu, float alpha)
{
    float *g = (float *)oracle_alloc((size_t)n * sizeof(float), 1); /* all +0 */
    for (uint32_t r = 0; r < nlists; r++) {
        for (uint64_t k = 0; k < count[r]; k++) {
            uint32_t j = idx[r][k];
            if (j < index_base || (uint64_t)(j - index_base) >= n)
                continue;
            g[j - index_base] = g[j - index_base] + val[r][k];
        }
    }
    for (uint64_t i = 0; i < n; i++) {
        float gi = g[i];
        if (nlists > 0)
            gi = gi / (float)nlists;
        float m = mu * momentum[i];
        m = m + gi;
        momentum[i] = m;
        float t = mu * m;
        t = t + gi;
        float step = alpha * t;
        theta[i] = theta[i] - step;
    }
    free(g);
    return 0;
}

/*
 * Index stream of one sorted list (App. H.2 "Index Encoding"; App. F.3 "Sparse
 * stream format": indices delta-encoded and varint-packed).
 *
 * The first index is stored as it is and every later one as its difference
 * from the previous index, d_0 = idx[0], d_k = idx[k] - idx[k-1] (indices
 * strictly ascending, so d_k >= 1 for k >= 1).  Each d_k is written as an
 * unsigned varint: 7-bit groups, least significant first, every byte but the
 * last of a number carrying 0x80.
 *
 * oracle_varint_encode writes bytes [0, out_capacity) of the stream and returns
 * its full length (the caller detects overflow as length > out_capacity).
 * oracle_varint_decode reads `nbytes` bytes and writes up to `max_out`
 * indices; it returns the number of indices in the stream, or -1 if the stream
 * ends inside a number.
 */
uint64_t oracle_varint_encode(const uint32_t *idx, uint64_t count, uint8_t *out,
                              uint64_t out_capacity)
{
    uint64_t pos = 0;
    for (uint64_t k = 0; k < count; k++) {
        uint32_t d = k == 0 ? idx[0] : idx[k] - idx[k - 1];
        for (;;) {
            uint8_t byte = (uint8_t)(d & 0x7F);
            d >>= 7;
            if (d != 0)
                byte |= 0x80;
            if (pos < out_capacity)
                out[pos] = byte;
            pos++;
            if (d == 0)
                break;
        }
    }
    return pos;
}

int64_t oracle_varint_decode(const uint8_t *in, uint64_t nbytes, uint32_t *out, uint64_t max_out)
{
    uint64_t count = 0, pos = 0;
    uint32_t prev = 0;
    while (pos < nbytes) {
        uint64_t d = 0;
        int shift = 0;
        for (;;) {
            if (pos >= nbytes)
                return -1;
            uint8_t byte = in[pos++];
            d |= (uint64_t)(byte & 0x7F) << shift;
            shift += 7;
            if (!(byte & 0x80))
                break;
        }
        uint32_t v = count == 0 ? (uint32_t)d : prev + (uint32_t)d;
        if (count < max_out)
            out[count] = v;
        prev = v;
        count++;
    }
    return (int64_t)count;
}

/* ------------------------------------------------------------------------
 * Weight-level integrity hash (App. J.4, "Weight-level integrity" and
 * "Deterministic hashing"; the hash h of Alg. 3 and of the sync protocol).
 *
 * The paper hashes the raw BF16 bit patterns of all parameters, concatenated
 * in a fixed order, with SHA-256.  The message here is that concatenation
 * as it sits in memory: each BF16 value as its two bytes, low byte first.
 *
 * A single SHA-256 over the whole stream is one long chain of compressions
 * and cannot be split across compute units, so the checksum is read as a
 * tree of SHA-256: the stream is cut into chunks of
 * `leaf_bytes` bytes (the last one may be shorter) and combined with the
 * Merkle Tree Hash of RFC 6962, Sec. 2.1:
 *     MTH({})      = SHA-256()                        (empty stream)
 *     MTH({c})     = SHA-256(0x00 || c)               (one chunk: leaf hash)
 *     MTH(D[0:n])  = SHA-256(0x01 || MTH(D[0:k]) || MTH(D[k:n])),
 *                    k = the largest power of two smaller than n.
 *
 * SHA-256 itself follows FIPS 180-4: padding (5.1.1), parsing into 512-bit
 * blocks (5.2.1), the initial hash value (5.3.3) and the computation (6.2.2).
 * Its constants are taken from their definitions rather than typed in: the
 * first 32 bits of the fractional parts of the square roots (initial hash
 * value) and cube roots (round constants) of the first primes, found here
 * with exact integer roots.
 * ------------------------------------------------------------------------ */

typedef struct {
    uint32_t k[64];
    uint32_t h0[8];
} sha_consts;

/* largest y with y^e <= v, by binary search over the bits of y (e = 2 or 3) */
static uint64_t iroot128(unsigned __int128 v, int e)
{
    uint64_t y = 0;
    for (int bit = 40; bit >= 0; bit--) {
        uint64_t t = y | ((uint64_t)1 << bit);
        unsigned __int128 p = (unsigned __int128)t * t;
        if (e == 3)
            p *= t;
        if (p <= v)
            y = t;
    }
    return y;
}

static void sha_make_consts(sha_consts *c)
{
    int found = 0;
    for (uint64_t p = 2; found < 64; p++) {
        int prime = 1;
        for (uint64_t d = 2; d * d <= p; d++)
            if (p % d == 0) {
                prime = 0;
                break;
            }
        if (!prime)
            continue;
        /* frac(cbrt(p)) * 2^32 = cbrt(p * 2^96) mod 2^32; likewise for sqrt */
        c->k[found] = (uint32_t)iroot128((unsigned __int128)p << 96, 3);
        if (found < 8)
            c->h0[found] = (uint32_t)iroot128((unsigned __int128)p << 64, 2);
        found++;
    }
}

static uint32_t rotr32(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

static void sha256_with(const sha_consts *c, const uint8_t *msg, uint64_t len, uint8_t out[32])
{
    /* 5.1.1: append the bit 1, zeros up to 448 mod 512 bits, and the 64-bit length */
    uint64_t padded = ((len + 8) / 64 + 1) * 64;
    uint8_t *m = oracle_alloc(padded, 1);
    if (len)
        memcpy(m, msg, len);
    m[len] = 0x80;
    uint64_t bits = len * 8;
    for (int i = 0; i < 8; i++)
        m[padded - 1 - i] = (uint8_t)(bits >> (8 * i));

    uint32_t H[8];
    memcpy(H, c->h0, sizeof H);
    for (uint64_t blk = 0; blk < padded / 64; blk++) {
        const uint8_t *M = m + 64 * blk;
        uint32_t W[64];
        for (int t = 0; t < 16; t++)
            W[t] = (uint32_t)M[4 * t] << 24 | (uint32_t)M[4 * t + 1] << 16 |
                   (uint32_t)M[4 * t + 2] << 8 | (uint32_t)M[4 * t + 3];
        for (int t = 16; t < 64; t++) {
            uint32_t s0 = rotr32(W[t - 15], 7) ^ rotr32(W[t - 15], 18) ^ (W[t - 15] >> 3);
            uint32_t s1 = rotr32(W[t - 2], 17) ^ rotr32(W[t - 2], 19) ^ (W[t - 2] >> 10);
            W[t] = s1 + W[t - 7] + s0 + W[t - 16];
        }
        uint32_t a = H[0], b = H[1], cc = H[2], d = H[3];
        uint32_t e = H[4], f = H[5], g = H[6], h = H[7];
        for (int t = 0; t < 64; t++) {
            uint32_t S1 = rotr32(e, 6) ^ rotr32(e, 11) ^ rotr32(e, 25);
            uint32_t ch = (e & f) ^ (~e & g);
            uint32_t T1 = h + S1 + ch + c->k[t] + W[t];
            uint32_t S0 = rotr32(a, 2) ^ rotr32(a, 13) ^ rotr32(a, 22);
            uint32_t maj = (a & b) ^ (a & cc) ^ (b & cc);
            uint32_t T2 = S0 + maj;
            h = g;
            g = f;
            f = e;
            e = d + T1;
            d = cc;
            cc = b;
            b = a;
            a = T1 + T2;
        }
        H[0] += a;
        H[1] += b;
        H[2] += cc;
        H[3] += d;
        H[4] += e;
        H[5] += f;
        H[6] += g;
        H[7] += h;
    }
    free(m);
    for (int i = 0; i < 8; i++)
        for (int j = 0; j < 4; j++)
            out[4 * i + j] = (uint8_t)(H[i] >> (24 - 8 * j));
}

void oracle_sha256(const uint8_t *msg, uint64_t len, uint8_t out[32])
{
    sha_consts c;
    sha_make_consts(&c);
    sha256_with(&c, msg, len, out);
}

/* leaf hash of RFC 6962: SHA-256 over the byte 0x00 followed by the chunk */
static void leaf_hash(const sha_consts *c, const uint8_t *chunk, uint64_t len, uint8_t out[32])
{
    uint8_t *buf = oracle_alloc(len + 1, 0);
    buf[0] = 0x00;
    if (len)
        memcpy(buf + 1, chunk, len);
    sha256_with(c, buf, len + 1, out);
    free(buf);
}

/* digests[i] = leaf hash of bytes [i*leaf_bytes, min((i+1)*leaf_bytes, nbytes)) */
void oracle_leaf_hashes(const uint8_t *stream, uint64_t nbytes, uint64_t leaf_bytes,
                        uint8_t *digests)
{
    sha_consts c;
    sha_make_consts(&c);
    uint64_t nleaves = (nbytes + leaf_bytes - 1) / leaf_bytes;
    for (uint64_t i = 0; i < nleaves; i++) {
        uint64_t lo = i * leaf_bytes;
        uint64_t len = nbytes - lo < leaf_bytes ? nbytes - lo : leaf_bytes;
        leaf_hash(&c, stream + lo, len, digests + 32 * i);
    }
}

/* MTH over the leaf digests d[lo, hi), hi - lo >= 1 */
static void mth(const sha_consts *c, const uint8_t *d, uint64_t lo, uint64_t hi, uint8_t out[32])
{
    uint64_t n = hi - lo;
    if (n == 1) {
        memcpy(out, d + 32 * lo, 32);
        return;
    }
    uint64_t k = 1;
    while (k * 2 < n)
        k *= 2;
    uint8_t node[65];
    node[0] = 0x01;
    mth(c, d, lo, lo + k, node + 1);
    mth(c, d, lo + k, hi, node + 33);
    sha256_with(c, node, sizeof node, out);
}

/* root of the tree over `nleaves` leaf digests (32 bytes each); no leaves:
 * the hash of the empty message */
void oracle_merkle_root(const uint8_t *digests, uint64_t nleaves, uint8_t root[32])
{
    sha_consts c;
    sha_make_consts(&c);
    if (nleaves == 0)
        sha256_with(&c, NULL, 0, root);
    else
        mth(&c, digests, 0, nleaves, root);
}

/* ------------------------------------------------------------------------
 * Lower-precision receivers (App. D): the compute view cast_D for
 * D = FP8 E4M3 and D = MXFP4, the patch of changed D-values, its apply, and
 * the compute-visibility gate G_D(theta, s) = {i : cast_D(theta_i) !=
 * cast_D(theta_i - s_i)} (App. D, its opening definition).
 *
 * Formats (OCP 8-bit floating point and OCP Microscaling v1.0, which App. D
 * names): FP8 E4M3 has bias 7, 3 mantissa bits, subnormals, no infinity,
 * NaN = S.1111.111, largest finite 448.  MXFP4 holds blocks of 32 consecutive
 * values of a tensor (the last block of a tensor may be shorter) as one E8M0
 * scale 2^E (byte E + 127) and 32 E2M1 codes (sign, 2 exponent bits, 1
 * mantissa bit: magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6), two codes per byte,
 * the even-indexed value in the low nibble.
 *
 * Readings where the paper is silent:
 *   - FP8 values carry a per-tensor FP32 scale: the receiver computes with
 *     y = fl32(x * inv_scale) cast to E4M3, rounded to nearest with ties to
 *     the even code, saturating to +-448 (also for +-inf); NaN -> 0x7F with
 *     the sign kept; the sign of a value rounding to zero is kept.
 *   - MXFP4: E = clamp(exponent field of the block's largest |x| - 129,
 *     -127, 127), i.e. floor(log2(amax)) - 2 for a normal amax (2 = the
 *     exponent of E2M1's largest value); zero and subnormal amax give -127,
 *     an infinite one 126.  A block holding a NaN gets scale byte 0xFF and
 *     all codes 0.  Each code is x / 2^E rounded to the nearest E2M1 value,
 *     ties to the even code, saturating to +-6, sign kept.
 *   - Compute view of an MXFP4 value = (its block's scale byte, its code);
 *     a patch entry carries both as (scale << 8) | code.
 * ------------------------------------------------------------------------ */

static double fp8_value(int c) /* c in 0..0x7E, magnitude */
{
    int e = c >> 3, m = c & 7;
    return e == 0 ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10);
}

uint8_t oracle_fp8_e4m3(float y)
{
    if (isnan(y))
        return (uint8_t)(0x7F | (signbit(y) ? 0x80 : 0));
    if (isinf(y)) /* saturating: the largest finite code */
        return (uint8_t)(0x7E | (signbit(y) ? 0x80 : 0));
    double a = fabs((double)y);
    int best = 0;
    double bd = a; /* distance to code 0 */
    for (int c = 1; c <= 0x7E; c++) {
        double d = fabs(a - fp8_value(c));
        if (d < bd || (d == bd && (c & 1) == 0)) {
            bd = d;
            best = c;
        }
    }
    return (uint8_t)(best | (signbit(y) ? 0x80 : 0));
}

double oracle_fp8_value(uint8_t c)
{
    if ((c & 0x7F) == 0x7F)
        return NAN;
    double v = fp8_value(c & 0x7F);
    return (c & 0x80) ? -v : v;
}

void oracle_cast_fp8(const float *x, uint8_t *out, uint64_t n, float inv_scale)
{
    for (uint64_t i = 0; i < n; i++) {
        float y = x[i] * inv_scale;
        out[i] = oracle_fp8_e4m3(y);
    }
}

static const double e2m1_mag[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

static uint8_t e2m1_code(double q) /* q finite or infinite, not NaN */
{
    if (isinf(q)) /* saturating: the largest magnitude, 6 */
        return (uint8_t)(7 | (signbit(q) ? 8 : 0));
    double a = fabs(q);
    int best = 0;
    double bd = a;
    for (int c = 1; c < 8; c++) {
        double d = fabs(a - e2m1_mag[c]);
        if (d < bd || (d == bd && (c & 1) == 0)) {
            bd = d;
            best = c;
        }
    }
    return (uint8_t)(best | (signbit(q) ? 8 : 0));
}

/* scale byte and codes of the block x[0..len) */
static uint8_t mx_block(const float *x, uint64_t len, uint8_t *codes)
{
    float amax = 0.0f;
    for (uint64_t i = 0; i < len; i++) {
        if (isnan(x[i])) {
            for (uint64_t j = 0; j < len; j++)
                codes[j] = 0;
            return 0xFF;
        }
        if (fabsf(x[i]) > amax)
            amax = fabsf(x[i]);
    }
    int ef = (int)((bits_from_float(amax) >> 23) & 0xFF);
    int E = ef - 129;
    if (E < -127)
        E = -127;
    if (E > 127)
        E = 127;
    for (uint64_t i = 0; i < len; i++)
        codes[i] = e2m1_code(ldexp((double)x[i], -E)); /* exact in double */
    return (uint8_t)(E + 127);
}

/* codes: (n + 1) / 2 bytes, scales: (n + 31) / 32 bytes */
void oracle_cast_mxfp4(const float *x, uint64_t n, uint8_t *codes, uint8_t *scales)
{
    uint8_t c[32];
    memset(codes, 0, (n + 1) / 2);
    for (uint64_t b = 0; b * 32 < n; b++) {
        uint64_t len = n - b * 32 < 32 ? n - b * 32 : 32;
        scales[b] = mx_block(x + b * 32, len, c);
        for (uint64_t i = 0; i < len; i++) {
            uint64_t k = b * 32 + i;
            codes[k / 2] |= (uint8_t)(c[i] << (4 * (k & 1)));
        }
    }
}

static uint8_t nibble(const uint8_t *codes, uint64_t k) { return (codes[k / 2] >> (4 * (k & 1))) & 0xF; }

/* Encode for an FP8 receiver: emit (index_base + i, code) wherever the code of
 * fl32(w_new * inv_scale) differs from snap[i]; capacity/count as oracle_encode. */
uint64_t oracle_encode_fp8(const float *w_new, const uint8_t *snap, uint64_t n, float inv_scale,
                           uint32_t index_base, uint32_t *idx, uint8_t *val, uint64_t capacity,
                           uint64_t count_in)
{
    uint64_t count = count_in;
    for (uint64_t i = 0; i < n; i++) {
        uint8_t c = oracle_fp8_e4m3(w_new[i] * inv_scale);
        if (c != snap[i]) {
            if (count < capacity) {
                idx[count] = index_base + (uint32_t)i;
                val[count] = c;
            }
            count++;
        }
    }
    return count;
}

/* Encode for an MXFP4 receiver: emit (index_base + i, (scale << 8) | code)
 * wherever the value's block scale or code differs from the snapshot's. */
uint64_t oracle_encode_mxfp4(const float *w_new, const uint8_t *snap_codes,
                             const uint8_t *snap_scales, uint64_t n, uint32_t index_base,
                             uint32_t *idx, uint16_t *val, uint64_t capacity, uint64_t count_in)
{
    uint64_t count = count_in;
    uint8_t c[32];
    for (uint64_t b = 0; b * 32 < n; b++) {
        uint64_t len = n - b * 32 < 32 ? n - b * 32 : 32;
        uint8_t s = mx_block(w_new + b * 32, len, c);
        for (uint64_t i = 0; i < len; i++) {
            uint64_t k = b * 32 + i;
            if (s != snap_scales[b] || c[i] != nibble(snap_codes, k)) {
                if (count < capacity) {
                    idx[count] = index_base + (uint32_t)k;
                    val[count] = (uint16_t)((s << 8) | c[i]);
                }
                count++;
            }
        }
    }
    return count;
}

/* Apply for an FP8 receiver: dst[idx[k] - index_base] = val[k], k in [begin, end);
 * returns the number of entries outside dst. */
uint64_t oracle_apply_fp8(uint8_t *dst, uint64_t n, const uint32_t *idx, const uint8_t *val,
                          uint64_t begin, uint64_t end, uint32_t index_base)
{
    uint64_t rejected = 0;
    for (uint64_t k = begin; k < end; k++) {
        uint64_t j = (uint64_t)idx[k] - index_base;
        if (idx[k] < index_base || j >= n) {
            rejected++;
            continue;
        }
        dst[j] = val[k];
    }
    return rejected;
}

/* Apply for an MXFP4 receiver: the entry's code into its nibble and its scale
 * into its block's scale byte. */
uint64_t oracle_apply_mxfp4(uint8_t *codes, uint8_t *scales, uint64_t n, const uint32_t *idx,
                            const uint16_t *val, uint64_t begin, uint64_t end, uint32_t index_base)
{
    uint64_t rejected = 0;
    for (uint64_t k = begin; k < end; k++) {
        uint64_t j = (uint64_t)idx[k] - index_base;
        if (idx[k] < index_base || j >= n) {
            rejected++;
            continue;
        }
        int sh = 4 * (int)(j & 1);
        codes[j / 2] = (uint8_t)((codes[j / 2] & ~(0xF << sh)) | ((val[k] & 0xF) << sh));
        scales[j / 32] = (uint8_t)(val[k] >> 8);
    }
    return rejected;
}

/* The PULSELoCo gate for a receiver computing in D (dtype 1 = FP8 E4M3 with
 * inv_scale, 2 = MXFP4): a = fl32(delta + e); keep i iff cast_D(theta)_i !=
 * cast_D(theta - a)_i (for MXFP4 the (scale, code) pairs, each vector with its
 * own block scales); emission, capacity and residual exactly as oracle_loco. */
uint64_t oracle_loco_gate_lp(int dtype, float inv_scale, const float *delta, float *residual,
                             uint64_t n, const float *theta, uint32_t index_base, uint32_t *idx,
                             float *val, uint64_t capacity, uint64_t count_in)
{
    float *a = oracle_alloc((size_t)n * sizeof(float), 0);
    float *after = oracle_alloc((size_t)n * sizeof(float), 0);
    uint8_t *keep = oracle_alloc(n, 0);
    for (uint64_t i = 0; i < n; i++) {
        a[i] = delta[i] + residual[i];
        after[i] = theta[i] - a[i];
    }
    if (dtype == 1) {
        for (uint64_t i = 0; i < n; i++)
            keep[i] = oracle_fp8_e4m3(theta[i] * inv_scale) != oracle_fp8_e4m3(after[i] * inv_scale);
    } else {
        uint8_t c0[32], c1[32];
        for (uint64_t b = 0; b * 32 < n; b++) {
            uint64_t len = n - b * 32 < 32 ? n - b * 32 : 32;
            uint8_t s0 = mx_block(theta + b * 32, len, c0);
            uint8_t s1 = mx_block(after + b * 32, len, c1);
            for (uint64_t i = 0; i < len; i++)
                keep[b * 32 + i] = s0 != s1 || c0[i] != c1[i];
        }
    }
    uint64_t count = count_in;
    for (uint64_t i = 0; i < n; i++) {
        if (keep[i] && count < capacity) {
            idx[count] = index_base + (uint32_t)i;
            val[count] = a[i];
            residual[i] = 0.0f;
        } else {
            residual[i] = a[i];
        }
        if (keep[i])
            count++;
    }
    free(a);
    free(after);
    free(keep);
    return count;
}

/* ------------------------------------------------------------------------
 * 2-D COO delta downcast of a patch's indices (App. H.2, step 4: downcast the
 * index types, uint8 row deltas and uint16 column deltas; App. H.4.1 "Type
 * downscaling"; the delta_coo_downscaled representation of App. H.4).
 *
 * A segment (one tensor, `cols` columns, entries ascending) is stored as its
 * first local index as it is (4 bytes, App. H.2 step 2) followed by one
 * (uint8 row field, uint16 column field) pair per later entry, row-major:
 *   same row as the previous entry:   (0, column - previous column)
 *   a later row, rows ahead = dr:     (dr, column + 1)
 * A jump of more than 255 rows is sent as (255, 0) escape pairs, each moving
 * 255 rows down without an entry, then the pair of the remaining 1..255 rows.
 * No entry yields (255, 0): a same-row pair has row field 0, a new-row pair a
 * column field >= 1.  Requires 1 <= cols <= 65535.  (The paper notes that
 * larger jumps are rare but does not say how they are kept lossless; the
 * escape pair is a reading of that gap.)
 * ------------------------------------------------------------------------ */

/* Pairs of all segments into drow/dcol (positions >= out_capacity are not
 * written); first[s] = the segment's first index (0 for an empty one),
 * seg_pairs[s] = where its pairs start.  Segment s holds entries
 * [seg_begin[s], seg_begin[s + 1]) (the last one up to nent).  Returns the
 * number of pairs. */
uint64_t oracle_coo_encode(const uint32_t *idx, uint64_t nent, const uint64_t *seg_begin,
                           uint32_t nseg, const uint32_t *cols, uint32_t *first, uint8_t *drow,
                           uint16_t *dcol, uint64_t out_capacity, uint64_t *seg_pairs)
{
    uint64_t np = 0;
    for (uint32_t s = 0; s < nseg; s++) {
        uint64_t b = seg_begin[s], e = s + 1 < nseg ? seg_begin[s + 1] : nent;
        uint64_t C = cols[s];
        seg_pairs[s] = np;
        first[s] = e > b ? idx[b] : 0;
        for (uint64_t k = b + 1; k < e; k++) {
            uint64_t r = idx[k] / C, c = idx[k] % C;
            uint64_t pr = idx[k - 1] / C, pc = idx[k - 1] % C;
            uint64_t dr = r - pr;
            if (dr == 0) {
                if (np < out_capacity) {
                    drow[np] = 0;
                    dcol[np] = (uint16_t)(c - pc);
                }
                np++;
                continue;
            }
            while (dr > 255) {
                if (np < out_capacity) {
                    drow[np] = 255;
                    dcol[np] = 0;
                }
                np++;
                dr -= 255;
            }
            if (np < out_capacity) {
                drow[np] = (uint8_t)dr;
                dcol[np] = (uint16_t)(c + 1);
            }
            np++;
        }
    }
    return np;
}

/* The indices back: entries of segment s go to out[seg_begin[s] ...].
 * Returns the number of entries, or -1 if a segment's pairs do not give
 * exactly its entry count or hold a pair no encoder writes. */
int64_t oracle_coo_decode(const uint8_t *drow, const uint16_t *dcol, uint64_t npairs,
                          const uint64_t *seg_pairs, const uint64_t *seg_begin, uint32_t nseg,
                          uint64_t nent, const uint32_t *cols, const uint32_t *first,
                          uint32_t *out)
{
    for (uint32_t s = 0; s < nseg; s++) {
        uint64_t b = seg_begin[s], e = s + 1 < nseg ? seg_begin[s + 1] : nent;
        uint64_t p0 = seg_pairs[s], p1 = s + 1 < nseg ? seg_pairs[s + 1] : npairs;
        uint64_t C = cols[s];
        if (e == b) {
            if (p1 != p0)
                return -1;
            continue;
        }
        uint64_t r = first[s] / C, c = first[s] % C, k = b;
        out[k++] = first[s];
        for (uint64_t q = p0; q < p1; q++) {
            if (drow[q] == 255 && dcol[q] == 0) {
                r += 255;
                continue;
            }
            if (drow[q] == 0) {
                if (dcol[q] == 0)
                    return -1;
                c += dcol[q];
            } else {
                if (dcol[q] == 0)
                    return -1;
                r += drow[q];
                c = dcol[q] - 1u;
            }
            if (k >= e)
                return -1;
            out[k++] = (uint32_t)(r * C + c);
        }
        if (k != e)
            return -1;
    }
    return (int64_t)nent;
}
