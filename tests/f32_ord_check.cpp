// Host check of the search library's order-preserving float32 cell mapping
// (f32_ord in boa_internal.h), which the index applies to float32 attribute
// columns and the kernels apply to each query's bounds. For every pair of
// non-NaN values a, b from a set of special and random floats:
// (a <= b) == (f32_ord(a) <= f32_ord(b)); both zeros map to 0; every NaN
// maps below the image of every non-NaN value. Exit status 0 when all hold.
#include "boa_internal.h"

#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>
#include <random>
#include <vector>

static uint32_t bits_of(float f)
{
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return u;
}

static float float_of(uint32_t u)
{
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

int main()
{
    std::vector<uint32_t> v;
    const float special[] = {0.0f, -0.0f, std::numeric_limits<float>::infinity(),
                             -std::numeric_limits<float>::infinity(), std::numeric_limits<float>::denorm_min(),
                             -std::numeric_limits<float>::denorm_min(), std::numeric_limits<float>::min(),
                             -std::numeric_limits<float>::min(), std::numeric_limits<float>::max(),
                             -std::numeric_limits<float>::max(), 1.0f, -1.0f, 0.5f, -0.5f, 1e-30f, -1e-30f};
    for (float f : special) v.push_back(bits_of(f));
    std::mt19937 rng(12345);
    std::uniform_int_distribution<uint32_t> any;
    while (v.size() < 2000) {
        const uint32_t u = any(rng);
        if (!std::isnan(float_of(u))) v.push_back(u);
    }
    const uint32_t nans[] = {0x7FC00000u, 0x7F800001u, 0xFFC00000u, 0xFFFFFFFFu, 0x7FFFFFFFu};
    long failures = 0;
    for (uint32_t a : v) {
        for (uint32_t b : v) {
            const bool fl = float_of(a) <= float_of(b);
            const bool in = boa::f32_ord(a) <= boa::f32_ord(b);
            if (fl != in && failures++ < 5)
                std::printf("order differs: %08x %08x float %d ord %d\n", a, b, (int)fl, (int)in);
        }
        for (uint32_t n : nans) {
            if (!(boa::f32_ord(n) < boa::f32_ord(a)) && failures++ < 5)
                std::printf("NaN %08x not below %08x\n", n, a);
        }
    }
    if (boa::f32_ord(0x00000000u) != 0 || boa::f32_ord(0x80000000u) != 0) {
        std::printf("zeros do not map to 0\n");
        ++failures;
    }
    std::printf("%ld failures over %zu values\n", failures, v.size());
    return failures == 0 ? 0 : 1;
}
