/*
 * MoE group-score oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * build, load or call this file.  The HIP library shares no code, header,
 * table or constant with it, and must never fall back to it.
 *
 * What it computes (the paper's running example, Motivation section, and the
 * figure of its source rewrite): the expert scores of a token are cut into
 * consecutive groups of G; the score of a group is the sum of its two largest
 * values, counted with multiplicity, so a maximum that occurs twice counts
 * twice.  The paper states that this equals the largest sum v_i + v_j over
 * two different positions i != j; the tests check the oracle against that
 * identity by brute force.
 *
 * Steps, per group: any NaN makes the score NaN (as a NaN-propagating top-2
 * does); otherwise take the maximum t1 and the first position p holding it,
 * then the maximum t2 over every position except p, and form t1 + t2.
 *
 * Precision: the two values are exactly representable in double and so is
 * their sum (two floats), and the sum is rounded once to float: the value of
 * an fp32 addition of the two stored scores.  For a bf16 result that float is
 * then rounded to bf16, to nearest with ties to even.  IEEE semantics hold for
 * infinities (+inf + -inf = NaN).  Build with -ffp-contract=off and no
 * fast-math.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* Round a float to the nearest bf16 (ties to even), returned as a float. */
static float round_to_bf16(float f)
{
    if (isnan(f))
        return f;
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    u += 0x7fffu + ((u >> 16) & 1u);
    u &= 0xffff0000u;
    memcpy(&f, &u, sizeof f);
    return f;
}

static double group_top2(const double *v, int64_t g, int bf16_out)
{
    for (int64_t i = 0; i < g; ++i)
        if (isnan(v[i]))
            return NAN;
    int64_t p = 0;
    for (int64_t i = 1; i < g; ++i)
        if (v[i] > v[p])
            p = i;
    double t2 = -INFINITY;
    for (int64_t i = 0; i < g; ++i)
        if (i != p && v[i] > t2)
            t2 = v[i];
    float s = (float)(v[p] + t2);
    return bf16_out ? (double)round_to_bf16(s) : (double)s;
}

/*
 * oracle_moe_group_top2_f64: scores is tokens x experts (row-major, values
 * already widened exactly from the stored dtype); out receives
 * tokens x (experts / group) scores.  Returns 0, or -1 when the group size
 * is below 2 or does not divide experts.
 */
int oracle_moe_group_top2_f64(const double *scores, double *out, int64_t tokens,
                              int64_t experts, int64_t group, int bf16_out)
{
    if (group < 2 || experts % group != 0)
        return -1;
    const int64_t ngroups = tokens * (experts / group);
    for (int64_t k = 0; k < ngroups; ++k)
        out[k] = group_top2(scores + k * group, group, bf16_out);
    return 0;
}
