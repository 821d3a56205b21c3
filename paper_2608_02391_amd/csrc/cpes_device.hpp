// cpes_device.hpp -- device functions of the CoPES hot path for gfx950:
// the Philox4x32-10 counter-based generator, the Box-Muller transform that
// turns its words into the Gaussian noise of Eq. (8), and bf16 storage.
//
// Seed replay (Sec. 3.3, Supp. A.8): the noise of every member is a pure
// function of (seed, position), so perturb, restore and update regenerate it in
// registers and nothing of size d is ever stored.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cpes {

// ----------------------------------------------------------------- Philox --
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies and xors, the key advancing by Weyl constants between
// rounds.  The key words come from kernel arguments, so the key schedule runs
// on the scalar unit.

constexpr uint32_t kPhiloxMulA = 0xD2511F53u;
constexpr uint32_t kPhiloxMulB = 0xCD9E8D57u;
constexpr uint32_t kWeylA = 0x9E3779B9u;
constexpr uint32_t kWeylB = 0xBB67AE85u;

struct Words4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ Words4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t pa = (uint64_t)kPhiloxMulA * c0;
        const uint64_t pb = (uint64_t)kPhiloxMulB * c2;
        const uint32_t n0 = (uint32_t)(pb >> 32) ^ c1 ^ k0;
        const uint32_t n2 = (uint32_t)(pa >> 32) ^ c3 ^ k1;
        c1 = (uint32_t)pb;
        c3 = (uint32_t)pa;
        c0 = n0;
        c2 = n2;
        k0 += kWeylA;
        k1 += kWeylB;
    }
    return Words4{c0, c1, c2, c3};
}

// Block q of stream (key, domain): counter (lo32 q, hi32 q, domain, 0).
__device__ __forceinline__ Words4 stream_block(uint32_t k0, uint32_t k1, uint32_t domain, uint64_t q)
{
    return philox4x32_10((uint32_t)q, (uint32_t)(q >> 32), domain, 0u, k0, k1);
}

// ------------------------------------------------------------ Box-Muller --
// A pair of words (a, b) gives two normals rho cos(theta), rho sin(theta) with
// rho = sqrt(-2 ln U(a)), theta = 2 pi U(b), U(x) = ((x >> 8) + 1) 2^-24.
// Both factors are evaluated in fp64 (full rate on CDNA4) to ~2^-44 relative
// error and their product is rounded once to fp32, so the result is the
// correctly rounded normal except within ~2^-20 of a rounding boundary.

// ln U for U = m 2^-24, m in [1, 2^24]: m = f 2^e with f in (1/sqrt2, sqrt2],
// ln U = (e - 24) ln 2 + 2 atanh((f - 1) / (f + 1)), the series truncated
// after s^15 (relative error < 4e-14 for |s| <= 3 - 2 sqrt2).
__device__ __forceinline__ double bm_radius(uint32_t a)
{
    const uint32_t m = (a >> 8) + 1u;
    const int lz = __clz((int)m);                 // m >= 1, so lz <= 31
    const uint32_t nm = m << lz;                  // top bit set: m = nm 2^-(lz)
    const int big = nm > 3037000499u ? 1 : 0;     // nm 2^-31 > sqrt(2)
    const int e = 31 - lz + big;                  // m = f 2^e
    const double f = __builtin_ldexp((double)nm, -31 - big);
    const double num = f - 1.0;                   // exact
    const double den = f + 1.0;                   // exact
    double r = __builtin_amdgcn_rcp(den);         // reciprocal estimate, refined twice
    double err = __builtin_fma(-den, r, 1.0);
    r = __builtin_fma(r, err, r);
    err = __builtin_fma(-den, r, 1.0);
    r = __builtin_fma(r, err, r);
    const double s = num * r;
    const double s2 = s * s;
    double p = 2.0 / 15.0;
    p = __builtin_fma(p, s2, 2.0 / 13.0);
    p = __builtin_fma(p, s2, 2.0 / 11.0);
    p = __builtin_fma(p, s2, 2.0 / 9.0);
    p = __builtin_fma(p, s2, 2.0 / 7.0);
    p = __builtin_fma(p, s2, 2.0 / 5.0);
    p = __builtin_fma(p, s2, 2.0 / 3.0);
    p = __builtin_fma(p, s2, 2.0);
    const double ln_f = s * p;
    const double ln_u = __builtin_fma((double)(e - 24), 0x1.62e42fefa39efp-1, ln_f);
    return __builtin_sqrt(-2.0 * ln_u);
}

// (cos, sin)(theta) for theta = pi m 2^-23, m = (b >> 8) + 1 in [1, 2^24].
// Quadrant and remainder are taken from m exactly; the remainder r (in units
// of 2^-23 half-turns) is folded to t in [0, 2^21] so that theta mod pi/2 is
// pi t 2^-23 or pi/2 minus it, and sin / cos(pi t 2^-23) are Taylor series in
// the integer t with coefficients (-1)^k pi^n / n! 2^(-23 n) (truncation
// error < 3e-14 relative on [0, pi/4]).  Exact zeros stay exact.
__device__ __forceinline__ void bm_angle(uint32_t b, double& c_out, double& s_out)
{
    const uint32_t m = (b >> 8) + 1u;
    const uint32_t quadrant = (m >> 22) & 3u;
    const uint32_t rem = m & 0x3FFFFFu;
    const bool fold = rem > (1u << 21);
    const double t = (double)(fold ? (1u << 22) - rem : rem);
    const double t2 = t * t;
    double sp = 0x1.e8f434d018d63p-311;
    sp = __builtin_fma(sp, t2, -0x1.e3074fde8871fp-261);
    sp = __builtin_fma(sp, t2, 0x1.50783487ee782p-211);
    sp = __builtin_fma(sp, t2, -0x1.32d2cce62bd86p-162);
    sp = __builtin_fma(sp, t2, 0x1.466bc6775aae2p-114);
    sp = __builtin_fma(sp, t2, -0x1.4abbce625be53p-67);
    sp = __builtin_fma(sp, t2, 0x1.921fb54442d18p-22);
    sp = sp * t;                                  // sin(pi t 2^-23)
    double cp = -0x1.b6e24f44b128fp-336;
    cp = __builtin_fma(cp, t2, 0x1.f9d38a3763cc3p-286);
    cp = __builtin_fma(cp, t2, -0x1.a6d1f2a204a8cp-236);
    cp = __builtin_fma(cp, t2, 0x1.e1f506891babbp-187);
    cp = __builtin_fma(cp, t2, -0x1.55d3c7e3cbffap-138);
    cp = __builtin_fma(cp, t2, 0x1.03c1f081b5ac4p-90);
    cp = __builtin_fma(cp, t2, -0x1.3bd3cc9be45dep-44);
    cp = __builtin_fma(cp, t2, 1.0);              // cos(pi t 2^-23)
    // Rotate by the quadrant: (c, s) = (C, S), (-S, C), (-C, -S), (S, -C) where
    // (C, S) = (cos, sin) of the remainder, i.e. (cp, sp) or, folded, (sp, cp).
    const bool take_sin = fold ^ ((quadrant & 1u) != 0u);
    const double mag_c = take_sin ? sp : cp;
    const double mag_s = take_sin ? cp : sp;
    c_out = (quadrant == 1u || quadrant == 2u) ? -mag_c : mag_c;
    s_out = (quadrant >= 2u) ? -mag_s : mag_s;
}

__device__ __forceinline__ void bm_pair(uint32_t a, uint32_t b, float& z_even, float& z_odd)
{
    const double rho = bm_radius(a);
    double c, s;
    bm_angle(b, c, s);
    z_even = (float)(rho * c);
    z_odd = (float)(rho * s);
}

// Four normals of block q: positions 4q .. 4q+3.
__device__ __forceinline__ void normals4(uint32_t k0, uint32_t k1, uint64_t q, float z[4])
{
    const Words4 x = stream_block(k0, k1, 0u, q);
    bm_pair(x.x, x.y, z[0], z[1]);
    bm_pair(x.z, x.w, z[2], z[3]);
}

// Eight normals of blocks q and q+1: positions 4q .. 4q+7.
__device__ __forceinline__ void normals8(uint32_t k0, uint32_t k1, uint64_t q, float z[8])
{
    const Words4 x = stream_block(k0, k1, 0u, q);
    const Words4 y = stream_block(k0, k1, 0u, q + 1u);
    bm_pair(x.x, x.y, z[0], z[1]);
    bm_pair(x.z, x.w, z[2], z[3]);
    bm_pair(y.x, y.y, z[4], z[5]);
    bm_pair(y.z, y.w, z[6], z[7]);
}

// ------------------------------------------------------------------ bf16 --

__device__ __forceinline__ float bf16_to_f32(uint16_t h)
{
    return __uint_as_float((uint32_t)h << 16);
}

// Round to nearest even; NaN stays a quiet NaN (gfx950 converts in hardware).
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    const __bf16 h = (__bf16)f;
    return __builtin_bit_cast(uint16_t, h);
}

}  // namespace cpes
