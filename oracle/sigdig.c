/*
 * Oracle (test infrastructure only): exact k-significant-digit quantiser of
 * binary32 history elements, the lossy history compression of Sec. 3
 * ("rounding ... with a smaller number of significant digits"; Table 1's
 * round-1 / round-2 rows).
 *
 * Reading taken where the paper is silent: rounding is to the nearest
 * k-significant-digit decimal, ties away from zero ("rounding up"); elements
 * lie in [-1, 1] (the paper notes this range under Table 1); magnitudes below
 * 1e-20 quantise to zero.
 *
 * Code layout (uint16): bit 15 = sign, bits 10..14 = e + 20, bits 0..9 = m,
 * for the value (-1)^sign * m * 10^(e - k + 1) with 10^(k-1) <= m < 10^k,
 * -20 <= e <= 0. Zero is the all-zero code.
 *
 * Arithmetic: |x| = M * 2^-s exactly (M < 2^24, s <= 149). Every comparison
 * and the rounding itself are done on integers in unsigned __int128, so no
 * floating-point rounding takes part in the decision.
 *
 * Plain, slow on purpose: e is found by stepping j = 0, 1, 2, ... rather than
 * estimated. Shares no code with the HIP library.
 */
#include <stdint.h>
#include <string.h>

typedef unsigned __int128 u128;

static u128 pow10_u128(int n)
{
    u128 r = 1;
    for (int i = 0; i < n; ++i) r *= 10;
    return r;
}

/* Returns 0 on success, 1 if some element is non-finite or |x| > 1. */
int oracle_sigdig_codes(const float *x, int64_t n, int k, uint16_t *out)
{
    if (k < 1 || k > 3) return 2;
    int bad = 0;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b;
        memcpy(&b, &x[i], 4);
        uint32_t neg = b >> 31;
        uint32_t mag = b & 0x7fffffffu;
        if (mag > 0x3f800000u) { bad = 1; out[i] = 0; continue; } /* |x|>1, inf, nan */
        uint32_t ex = mag >> 23, fr = mag & 0x7fffffu;
        uint64_t M = ex ? (fr | 0x800000u) : fr;
        int s = ex ? 150 - (int)ex : 149;              /* |x| = M * 2^-s */
        if (M == 0 || s >= 128) { out[i] = 0; continue; } /* zero or < 2^-104 */
        u128 two_s = (u128)1 << s;
        /* |x| < 1e-20  <=>  M * 10^20 < 2^s */
        if ((u128)M * pow10_u128(20) < two_s) { out[i] = 0; continue; }
        /* e = floor(log10 |x|) = -j for the smallest j >= 0 with M*10^j >= 2^s */
        int j = 0;
        while ((u128)M * pow10_u128(j) < two_s) ++j;
        int e = -j;
        int p = k - 1 + j;                               /* |x| * 10^p in [10^(k-1), 10^k) */
        /* m = floor(M * 10^p / 2^s + 1/2): nearest integer, ties away from zero */
        u128 m = ((u128)M * pow10_u128(p) + (two_s >> 1)) >> s;
        if (m == pow10_u128(k)) { m = pow10_u128(k - 1); e += 1; }
        out[i] = (uint16_t)((neg << 15) | ((uint32_t)(e + 20) << 10) | (uint32_t)m);
    }
    return bad;
}
