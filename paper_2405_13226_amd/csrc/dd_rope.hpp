// dd_rope.hpp -- rotary position embedding on the device (arXiv 2405.13226,
// Sec. 3, "Positional encoding"): components (2j, 2j+1) of a head vector are
// rotated by the angle pos * base^(-2j/D).
//
// The per-pair frequencies base^(-2j/D) are formed in double precision from
// six powers of rho = base^(-2/D) that the host computes and passes by value
// (rope_theta_j: every kernel forms theta_j with the same operations, so a
// rotation done in one kernel is bit-identical to the same rotation done in
// another).  An angle pos * theta (up to ~1.6e4 rad) is formed in double and
// reduced to a fraction of a turn before the fp32 sine and cosine, so its
// error stays at the fp32 rounding of the reduced angle rather than growing
// with the position.
#pragma once

#include "dd_device.hpp"

namespace dd {

// Sine and cosine of pos * theta: the angle in turns (a / 2pi) is formed in
// double and reduced to its fractional part in [-1/2, 1/2]; the hardware
// sine and cosine take their argument in turns.
__device__ __forceinline__ void rope_sincos(double theta, int pos, float &s, float &c)
{
    const double turns = static_cast<double>(pos) * theta * 0.15915494309189533577;
    const float t = static_cast<float>(turns - rint(turns));
    s = __builtin_amdgcn_sinf(t);
    c = __builtin_amdgcn_cosf(t);
}

// (x0, x1) rotated by the angle whose sine and cosine are s, c; the transposed
// rotation when INV.
template <bool INV>
__device__ __forceinline__ void rope_pair(float &x0, float &x1, float s, float c)
{
    const float y0 = INV ? fmaf(x0, c, x1 * s) : fmaf(x0, c, -x1 * s);
    const float y1 = INV ? fmaf(x1, c, -x0 * s) : fmaf(x0, s, x1 * c);
    x0 = y0;
    x1 = y1;
}

// Position of row-local token p of row b for mode 1 (row positions) or 2
// (positions from the start of the token's document inside the row).
__device__ __forceinline__ int rope_position(int b, int L, int p, const int32_t *__restrict__ cu,
                                             int n_docs, int mode)
{
    if (mode != 2)
        return p;
    int ds, de;
    doc_span(b, L, p, cu, n_docs, ds, de);
    return p - ds;
}

// Frequencies, with rho = base^(-2/D): p0..p3 = rho^0..rho^3, r4 = rho^4,
// r16 = rho^16 (six doubles instead of the full table keep the kernels'
// scalar registers free for their main loops).
struct RopeEpi {
    double p0, p1, p2, p3, r4, r16;
};

// (host; defined in dd_rope.hip)
RopeEpi rope_epi(double base, int D);

// theta_j = rho^(j mod 4) * (r16^(j / 16) * r4^((j / 4) mod 4)), the powers
// of r16 and r4 multiplied in that order starting from 1.  Every rotation
// in the library forms its frequencies this way.
__device__ __forceinline__ double rope_theta_j(const RopeEpi &re, int j)
{
    double s = 1.0;
    for (int i = 0; i < (j >> 4); ++i)
        s *= re.r16;
    for (int i = 0; i < ((j >> 2) & 3); ++i)
        s *= re.r4;
    const int c = j & 3;
    const double p = c == 0 ? re.p0 : c == 1 ? re.p1 : c == 2 ? re.p2 : re.p3;
    return p * s;
}

// Transposed rotation of the fp32 gradient rows a lane holds in the C layout
// of a 32x32 product (rows = head dims): acc[db][4*rg + e] is dim
// db*32 + 8*rg + 4*g + e, so pairs (e, e+1) for e = 0, 2 are in-lane and
// pair j = 16*db + 4*rg + 2*g + e/2 has theta_j = p[2g + e/2] * r16^db * r4^rg
// (rope_theta_j's operations, stepped across the registers).
template <int DB>
__device__ __forceinline__ void rope_unrotate_acc(f32x16 (&acc)[DB], const RopeEpi &re, int pos,
                                                  int g)
{
    const double base0 = g ? re.p2 : re.p0, base1 = g ? re.p3 : re.p1;
    double step_db = 1.0;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        double step = step_db;
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
#pragma unroll
            for (int pe = 0; pe < 2; ++pe) {
                float s, c;
                rope_sincos((pe ? base1 : base0) * step, pos, s, c);
                float x0 = acc[db][4 * rg + 2 * pe], x1 = acc[db][4 * rg + 2 * pe + 1];
                rope_pair<true>(x0, x1, s, c);
                acc[db][4 * rg + 2 * pe] = x0;
                acc[db][4 * rg + 2 * pe + 1] = x1;
            }
            step *= re.r4;
        }
        step_db *= re.r16;
    }
}

}  // namespace dd
