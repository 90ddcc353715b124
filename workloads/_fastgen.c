/*
 * Fast fill of synthetic prompt tokens (input generation only; no part of
 * the routing method).
 *
 * Random tokens come from PCG32 (O'Neill 2014, XSH-RR output of a 64-bit
 * LCG), one independent stream per 2^22-token chunk so the result does not
 * depend on the number of threads; a token is (u32 * vocab) >> 32.
 */
#include <stdint.h>
#include <string.h>

#define CHUNK (1LL << 22)

static uint32_t pcg32(uint64_t *state, uint64_t inc)
{
    uint64_t old = *state;
    *state = old * 6364136223846793005ULL + inc;
    uint32_t xorshifted = (uint32_t)(((old >> 18u) ^ old) >> 27u);
    uint32_t rot = (uint32_t)(old >> 59u);
    return (xorshifted >> rot) | (xorshifted << ((32u - rot) & 31u));
}

void fg_uniform_tokens(int32_t *out, int64_t n, uint32_t vocab, uint64_t seed)
{
    int64_t nchunks = (n + CHUNK - 1) / CHUNK;
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < nchunks; c++) {
        uint64_t inc = ((seed << 1) ^ ((uint64_t)c << 20)) | 1ULL;
        uint64_t st = 0;
        pcg32(&st, inc);
        st += seed ^ (0x853c49e6748fea9bULL + (uint64_t)c);
        pcg32(&st, inc);
        int64_t lo = c * CHUNK, hi = lo + CHUNK < n ? lo + CHUNK : n;
        for (int64_t i = lo; i < hi; i++)
            out[i] = (int32_t)(((uint64_t)pcg32(&st, inc) * vocab) >> 32);
    }
}

/* Request r's first shared[r] tokens become template tpl[r]'s first tokens. */
void fg_copy_prefixes(int32_t *tok, const int64_t *off, const int64_t *tpl, const int64_t *shared,
                      const int32_t *ttok, const int64_t *toff, int64_t n)
{
#pragma omp parallel for schedule(dynamic, 4096)
    for (int64_t r = 0; r < n; r++)
        if (shared[r] > 0)
            memcpy(tok + off[r], ttok + toff[tpl[r]], (size_t)shared[r] * sizeof(int32_t));
}
