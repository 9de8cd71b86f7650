/*
 * Seeded synthetic prompt text for the DriftSched admission workloads.
 *
 * Input synthesis only: this file holds no stage arithmetic. Prompt i gets
 * words[i] words of 1..12 random lowercase letters, separated by runs of
 * 1..3 characters drawn from {space, tab, newline}, with no leading or
 * trailing separator. With nonascii_p > 0 each letter is replaced, with that
 * probability, by one of a fixed set of two- and three-byte UTF-8 letters.
 *
 * Randomness: one SplitMix64 stream per prompt, started from a hash of
 * (seed, prompt index), so prompts can be generated in parallel and the
 * result does not depend on the number of threads. Integer draws in [0, k)
 * take the high 32 bits of a 32x32-bit product (multiply-shift reduction).
 */
#include <stdint.h>
#include <string.h>

static const uint8_t SEP[3] = { ' ', '\t', '\n' };

/* UTF-8 of: A-ring, a-grave, micro, Cyrillic Er, copyright, lambda,
 * a-stroke, hiragana a, CJK one, hyphen U+2010, A-ring-below, ideographic
 * number zero. None is whitespace; several share leading bytes with
 * multi-byte whitespace. */
static const uint8_t POOL[12][3] = {
    {0xC3, 0x85, 0}, {0xC3, 0xA0, 0}, {0xC2, 0xB5, 0}, {0xD0, 0xA0, 0},
    {0xC2, 0xA9, 0}, {0xCE, 0xBB, 0}, {0xE2, 0xB1, 0xA5}, {0xE3, 0x81, 0x82},
    {0xE4, 0xB8, 0x80}, {0xE2, 0x80, 0x90}, {0xE1, 0xB8, 0x80}, {0xE3, 0x80, 0x87},
};
static const uint8_t POOL_LEN[12] = { 2, 2, 2, 2, 2, 2, 3, 3, 3, 3, 3, 3 };

typedef struct { uint64_t s; uint64_t buf; int have; } rng_t;

static inline uint64_t sm64(uint64_t *s)
{
    uint64_t z = (*s += 0x9E3779B97F4A7C15ULL);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint32_t next32(rng_t *r)
{
    if (r->have) { r->have = 0; return (uint32_t)(r->buf >> 32); }
    r->buf = sm64(&r->s);
    r->have = 1;
    return (uint32_t)r->buf;
}

static inline uint32_t below(rng_t *r, uint32_t k)
{
    return (uint32_t)(((uint64_t)next32(r) * k) >> 32);
}

static void start(rng_t *r, uint64_t seed, uint64_t i)
{
    uint64_t s = seed * 0xD1B54A32D192ED03ULL + 0x8CB92BA72F3D8DD7ULL;
    r->s = s ^ (i * 0x9E3779B97F4A7C15ULL);
    (void)sm64(&r->s);
    r->have = 0;
}

/* Generate one prompt; out may be NULL (length only). Returns its bytes. */
static uint64_t prompt(uint64_t seed, uint64_t i, uint32_t nwords, uint32_t na_thresh,
                       int nonascii, uint8_t *out)
{
    rng_t r;
    start(&r, seed, i);
    uint64_t p = 0;
    for (uint32_t w = 0; w < nwords; w++) {
        uint32_t len = 1 + below(&r, 12);
        for (uint32_t k = 0; k < len; k++) {
            uint32_t letter = below(&r, 26);
            if (nonascii && next32(&r) < na_thresh) {
                uint32_t c = below(&r, 12);
                if (out) memcpy(out + p, POOL[c], POOL_LEN[c]);
                p += POOL_LEN[c];
            } else {
                if (out) out[p] = (uint8_t)('a' + letter);
                p += 1;
            }
        }
        if (w + 1 < nwords) {
            uint32_t ns = 1 + below(&r, 3);
            for (uint32_t k = 0; k < ns; k++) {
                uint32_t c = below(&r, 3);
                if (out) out[p] = SEP[c];
                p += 1;
            }
        }
    }
    return p;
}

/*
 * Pass 1 (out == NULL): lengths[i] = bytes of prompt i. Returns the total.
 * Pass 2 (out != NULL): fills out at offsets[i] (prefix sums of pass 1).
 */
int64_t synth_text(uint64_t seed, const uint32_t *words, uint64_t n, double nonascii_p,
                   uint8_t *out, const uint64_t *offsets, uint64_t *lengths)
{
    int nonascii = nonascii_p > 0.0;
    double t = nonascii_p * 4294967296.0;
    uint32_t thresh = t >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)t;
    int64_t total = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(+ : total)
    for (int64_t i = 0; i < (int64_t)n; i++) {
        if (out) {
            (void)prompt(seed, (uint64_t)i, words[i], thresh, nonascii, out + offsets[i]);
        } else {
            uint64_t l = prompt(seed, (uint64_t)i, words[i], thresh, nonascii, NULL);
            lengths[i] = l;
            total += (int64_t)l;
        }
    }
    return total;
}
