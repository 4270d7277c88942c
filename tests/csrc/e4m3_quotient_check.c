/* The append's e4m3 quantisation takes RN(x / s) for a scale s shared by a
 * (block, head) tile without dividing per value: r = RN(1/s), q0 = RN(x r),
 * e = fma(-q0, s, x), q1 = fma(e, r, q0) (Markstein's correction), with q0
 * kept where |q0| >= 512 (every such value saturates) and q0's sign; scales
 * outside [2^-100, 2^100] divide.  This program checks, for every finite
 * bf16 x and the scales s = fp32(b / 448) of every STRIDE-th positive finite
 * bf16 b (plus s = 1), that the e4m3 code of that quotient equals the code of
 * the correctly rounded quotient.  The code is computed by a plain search
 * for the nearest e4m3 value (ties to the even code, saturating at 448).
 * Prints the number of pairs and of mismatches. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float bf16(uint32_t b) { uint32_t u = b << 16; float f; memcpy(&f, &u, 4); return f; }

static float value(int c) {   /* positive e4m3 code c in 0..0x7E */
    int e = c >> 3, m = c & 7;
    return e == 0 ? ldexpf((float)m, -9) : ldexpf(1.0f + m / 8.0f, e - 7);
}

static int table_ready = 0;
static float vals[0x7F];

static int encode(float y) {
    if (isnan(y)) return 0x7F;
    int sign = signbit(y) ? 0x80 : 0;
    float a = fabsf(y);
    if (a >= 448.0f) return sign | 0x7E;
    if (!table_ready) { for (int c = 0; c <= 0x7E; ++c) vals[c] = value(c); table_ready = 1; }
    /* binary search for the first value >= a, then pick the nearer neighbour */
    int lo = 0, hi = 0x7E;
    while (lo < hi) { int mid = (lo + hi) / 2; if (vals[mid] >= a) hi = mid; else lo = mid + 1; }
    int best = lo;
    if (lo > 0) {
        float dl = a - vals[lo - 1], dh = vals[lo] - a;
        if (dl < dh || (dl == dh && ((lo - 1) & 1) == 0)) best = lo - 1;
    }
    return sign | best;
}

static float quotient(float x, float s, float r) {
    if (!(s >= 0x1p-100f && s <= 0x1p100f)) return x / s;
    const float q0 = x * r;
    const float e = fmaf(-q0, s, x);
    const float q1 = fmaf(e, r, q0);
    return copysignf(fabsf(q0) < 512.0f ? q1 : q0, q0);
}

int main(int argc, char **argv) {
    const int stride = argc > 1 ? atoi(argv[1]) : 1;
    static float xs[65536];
    int nx = 0;
    for (uint32_t b = 0; b < 65536; ++b) { float x = bf16(b); if (isfinite(x)) xs[nx++] = x; }
    /* scales: every stride-th positive finite bf16 b as b / 448, the last
     * one, those next to the edges of the fast range, and 1 */
    static float scales[0x8000 + 64];
    int ns = 0;
    for (uint32_t sb = 1; sb < 0x7F80; sb += stride) scales[ns++] = (float)((double)bf16(sb) / 448.0);
    scales[ns++] = (float)((double)bf16(0x7F7F) / 448.0);
    for (int k = -2; k <= 2; ++k) {
        scales[ns++] = nextafterf(0x1p-100f, k < 0 ? 0.0f : 1.0f) * (k == 0 ? 0.0f : 1.0f) + (k == 0 ? 0x1p-100f : 0.0f);
        scales[ns++] = nextafterf(0x1p100f, k < 0 ? 0.0f : INFINITY) * (k == 0 ? 0.0f : 1.0f) + (k == 0 ? 0x1p100f : 0.0f);
    }
    scales[ns++] = 1.0f;
    long long pairs = 0, bad = 0;
    for (int si = 0; si < ns; ++si) {
        const float s = scales[si];
        if (!(s > 0.0f) || !isfinite(s)) continue;
        const float r = 1.0f / s;
        for (int i = 0; i < nx; ++i) {
            const float x = xs[i];
            const float ref = (float)((double)x / (double)s);
            ++pairs;
            if (encode(quotient(x, s, r)) != encode(ref)) {
                if (bad < 5) printf("x=%a s=%a\n", x, s);
                ++bad;
            }
        }
    }
    printf("%lld %lld\n", pairs, bad);
    return 0;
}
