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

#include "cpes_log_table.hpp"

namespace cpes {

// ----------------------------------------------------------------- Philox --
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies and xors, the key advancing by Weyl constants between
// rounds.  The key words come from kernel arguments, so the key schedule runs
// on the scalar unit; each three-way xor is one v_bitop3_b32 (truth table
// 0x96) on gfx950.

constexpr uint32_t kPhiloxMulA = 0xD2511F53u;
constexpr uint32_t kPhiloxMulB = 0xCD9E8D57u;
constexpr uint32_t kWeylA = 0x9E3779B9u;
constexpr uint32_t kWeylB = 0xBB67AE85u;

struct Words4 {
    uint32_t x, y, z, w;
};

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ Words4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t pa = (uint64_t)kPhiloxMulA * c0;
        const uint64_t pb = (uint64_t)kPhiloxMulB * c2;
        const uint32_t n0 = xor3((uint32_t)(pb >> 32), c1, k0);
        const uint32_t n2 = xor3((uint32_t)(pa >> 32), c3, k1);
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
// Both factors are evaluated in fp64 (full rate on CDNA4) to ~2^-41 relative
// error and their product is rounded once to fp32, so the result is the
// correctly rounded normal except within ~2^-17 relative of a rounding
// boundary (and always within one fp32 ulp of it).
//
// The angle polynomials are near-minimax fits (relative error) computed
// offline with 120-bit arithmetic; the error of each evaluation is stated.

// L = -2 ln U for U = m 2^-24, m in [1, 2^24], table-driven (Tang's method):
// mn = m << lz is m normalised to [2^31, 2^32); entry i = bits 30..23 of mn
// holds inv_i ~ 2^-31 / c_i and B_i = -2 ln c_i for a point c_i of that
// 1/256-wide mantissa interval (cpes_log_table.hpp).  Then
//   r = mn inv_i - 1  (one fma, |r| <= 2^-8),
//   L = (lz - 7) 2 ln 2 + B_i - 2 ln(1 + r),
// with -2 ln(1 + r) = r q(r), q of degree 4 (Taylor).  Relative error at
// most 2^-46.5 over all 2^24 inputs; U = 1 gives L = 0 exactly.  The table
// lives in LDS (`lt`), staged once per workgroup by stage_log_table().
__device__ __forceinline__ double bm_log_term(uint32_t a, const LogEntry* lt)
{
    const uint32_t m7 = ((a >> 8) + 1u) << 7;             // m 2^7 <= 2^31
    const uint32_t e = (uint32_t)__builtin_clz(m7);        // lz - 7, in [0, 24]
    const uint32_t mn = m7 << e;
    static_assert(sizeof(LogEntry) == 16, "16-byte table entries");
    const uint32_t byte_off = (mn >> (27 - kLogTableBits)) & ((kLogTableSize - 1) << 4);   // entry * 16
    const LogEntry t = *reinterpret_cast<const LogEntry*>(reinterpret_cast<const char*>(lt) + byte_off);
    const double r = __builtin_fma((double)mn, t.inv, -1.0);
    const double base = __builtin_fma((double)e, kTwoLn2, t.b);
    double q = -0x1.999999999999ap-2;                      // -2/5
    q = __builtin_fma(q, r, 0.5);
    q = __builtin_fma(q, r, -0x1.5555555555555p-1);        // -2/3
    q = __builtin_fma(q, r, 1.0);
    q = __builtin_fma(q, r, -2.0);
    return __builtin_fma(r, q, base);
}

// Copy the log table into LDS; every thread of the workgroup must call it
// (it ends with a barrier).
__device__ __forceinline__ const LogEntry* stage_log_table()
{
    __shared__ LogEntry lt[kLogTableSize];
    for (int i = threadIdx.x; i < kLogTableSize; i += blockDim.x) lt[i] = kLogTable[i];
    __syncthreads();
    return lt;
}

// rho = sqrt(L): hardware reciprocal square root (2^-24) and one Goldschmidt
// step (2^-47).  The 2^-400 bias only keeps the estimate finite at L = 0
// (it vanishes in rounding for every L > 0), so rho(-0) = -0 like sqrt.
__device__ __forceinline__ double bm_sqrt(double L)
{
    const double y = __builtin_amdgcn_rsq(L + 0x1p-400);
    const double g = L * y;
    const double h = 0.5 * y;
    return __builtin_fma(g, __builtin_fma(-g, h, 0.5), g);
}

__device__ __forceinline__ double bm_radius(uint32_t a, const LogEntry* lt)
{
    return bm_sqrt(bm_log_term(a, lt));
}

// Angle theta = pi m 2^-23, m = (b >> 8) + 1 in [1, 2^24].  Quadrant and
// remainder come from m exactly; the remainder rem (units of 2^-23
// half-turns) is folded to t = min(rem, 2^22 - rem) in [0, 2^21], and
// sp = sin(pi t 2^-23) (degree-5 odd-power fit, 2^-47), cp = cos(pi t 2^-23)
// (degree 5 in t^2 with constant 1, 2^-41.6).  sp and cp are magnitudes; the
// caller places them by quadrant: (cos, sin) = (C, S), (-S, C), (-C, -S),
// (S, -C), with (C, S) = (cp, sp), or (sp, cp) when folded.
struct AngleParts {
    double sp, cp;
    bool take_sin;       // cos theta = +-sp (and sin theta = +-cp)
    uint32_t cos_sign;   // bit 31: sign of cos theta (other bits are not used)
    uint32_t sin_sign;   // bit 31: sign of sin theta (other bits are not used)
};

__device__ __forceinline__ AngleParts bm_angle_parts(uint32_t b)
{
    // s8 = (m << 8) mod 2^32, m = (b >> 8) + 1: adding 0x100 to b cannot carry
    // out of its low byte, so bits 8..31 of s8 are m's bits 0..23 (m = 2^24
    // wraps to 0, the same angle); bit 31 of s8 is then the sign of sin theta.
    const uint32_t s8 = b + 0x100u;
    const uint32_t rem = (s8 >> 8) & 0x3FFFFFu;             // m mod 2^22
    const bool fold = rem > (1u << 21);
    const double t = (double)(fold ? (1u << 22) - rem : rem);
    const double t2 = t * t;
    double sp = -0x1.dd4e53cfc3ebep-261;
    sp = __builtin_fma(sp, t2, 0x1.5071bed3ae526p-211);
    sp = __builtin_fma(sp, t2, -0x1.32d2c62989f77p-162);
    sp = __builtin_fma(sp, t2, 0x1.466bc670fd116p-114);
    sp = __builtin_fma(sp, t2, -0x1.4abbce62577b8p-67);
    sp = __builtin_fma(sp, t2, 0x1.921fb54442cf8p-22);
    sp = sp * t;
    double cp = -0x1.a1e54d0df20f1p-236;
    cp = __builtin_fma(cp, t2, 0x1.e1ec6573b80dcp-187);
    cp = __builtin_fma(cp, t2, -0x1.55d3c1b49a018p-138);
    cp = __builtin_fma(cp, t2, 0x1.03c1f07e99c51p-90);
    cp = __builtin_fma(cp, t2, -0x1.3bd3cc9be35d0p-44);
    cp = __builtin_fma(cp, t2, 1.0);
    AngleParts r;
    r.sp = sp;
    r.cp = cp;
    r.take_sin = fold ^ (((s8 >> 30) & 1u) != 0u);          // odd quadrant (bit 22 of m) swaps the roles
    r.cos_sign = s8 + 0x40000000u;                          // bit 31: quadrant 1 or 2
    r.sin_sign = s8;                                        // bit 31: quadrant 2 or 3
    return r;
}

// (cos, sin)(theta) as fp64 values (test hook).
__device__ __forceinline__ void bm_angle(uint32_t b, double& c_out, double& s_out)
{
    const AngleParts p = bm_angle_parts(b);
    const double mc = p.take_sin ? p.sp : p.cp;
    const double ms = p.take_sin ? p.cp : p.sp;
    c_out = (p.cos_sign & 0x80000000u) ? -mc : mc;
    s_out = (p.sin_sign & 0x80000000u) ? -ms : ms;
}

// z with its sign flipped where bit 31 of `sign` is set: one v_bitop3_b32
// computing z ^ (sign & 0x80000000) (truth table 0x78 for src0 ^ (src1 & src2)).
__device__ __forceinline__ float xor_sign(float z, uint32_t sign)
{
    return __uint_as_float(__builtin_amdgcn_bitop3_b32(__float_as_uint(z), sign, 0x80000000u, 0x78));
}

// Two normals of the pair (a, b): z_even = fp32(rho cos theta), z_odd =
// fp32(rho sin theta).  The products are formed from the magnitudes and the
// quadrant's swap and signs are applied to the fp32 results, which is exact
// (negation commutes with multiplication and rounding).
__device__ __forceinline__ void bm_pair(uint32_t a, uint32_t b, const LogEntry* lt, float& z_even, float& z_odd)
{
    const double rho = bm_radius(a, lt);
    const AngleParts p = bm_angle_parts(b);
    const float zc = (float)(rho * p.cp);
    const float zs = (float)(rho * p.sp);
    const float me = p.take_sin ? zs : zc;
    const float mo = p.take_sin ? zc : zs;
    z_even = xor_sign(me, p.cos_sign);
    z_odd = xor_sign(mo, p.sin_sign);
}

// Four normals of block q: positions 4q .. 4q+3 (domain 0 is the noise).
__device__ __forceinline__ void normals4(uint32_t k0, uint32_t k1, uint64_t q, const LogEntry* lt, float z[4],
                                         uint32_t domain = 0u)
{
    const Words4 x = stream_block(k0, k1, domain, q);
    bm_pair(x.x, x.y, lt, z[0], z[1]);
    bm_pair(x.z, x.w, lt, z[2], z[3]);
}

// Eight normals of blocks q and q+1: positions 4q .. 4q+7.
__device__ __forceinline__ void normals8(uint32_t k0, uint32_t k1, uint64_t q, const LogEntry* lt, float z[8],
                                         uint32_t domain = 0u)
{
    const Words4 x = stream_block(k0, k1, domain, q);
    const Words4 y = stream_block(k0, k1, domain, q + 1u);
    bm_pair(x.x, x.y, lt, z[0], z[1]);
    bm_pair(x.z, x.w, lt, z[2], z[3]);
    bm_pair(y.x, y.y, lt, z[4], z[5]);
    bm_pair(y.z, y.w, lt, z[6], z[7]);
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
