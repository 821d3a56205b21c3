/*
 * cpes_oracle.c -- plain CPU oracle for the CoPES parameter-space hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or constant generator with the GPU library; both sides are
 * written independently from the paper ("Cooperative Coevolution for
 * Resource-Constrained Agentic LLM Post-Training", arXiv 2608.02391) and from
 * the published definitions of the generators named below.
 *
 * Arithmetic: every floating-point step is written out in IEEE double (the
 * paper fixes no precision for these steps) and rounded once to the storage
 * type.  The one exception is the perturbation itself, which is defined as a
 * single fp32 fused multiply-add (fmaf is correctly rounded in glibc).  The
 * file is compiled without fast-math and with -ffp-contract=off so that the
 * compiler fuses nothing the text does not say.  OpenMP only splits loops whose
 * iterations are independent; results do not depend on the thread count.
 *
 * Readings of the paper where it is silent (the generator, the normal
 * transform, the partition algorithm, rank normalisation) are marked
 * "reading:" below.
 *
 * Parity status: every function here is pinned by the CPU tests (published
 * generator implementations, closed forms, brute force on tiny inputs,
 * statistics).  The paper's own noise stream is unknowable (its generator is
 * unspecified), so equality with the paper's training runs is parity unpinned.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#include "cpes_oracle.h"

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as     */
/* easy as 1, 2, 3", SC'11).  The paper represents each perturbation by a     */
/* seed and regenerates it during the update (Sec. 3.3, Supp. A.8 "Seed       */
/* Replay and Chunking") but names no generator.                              */
/* reading: a counter-based generator, Philox4x32 with 10 rounds.             */
/* ------------------------------------------------------------------------- */

#define PHILOX_M0 0xD2511F53u /* multiplier applied to counter word 0 */
#define PHILOX_M1 0xCD9E8D57u /* multiplier applied to counter word 2 */
#define PHILOX_W0 0x9E3779B9u /* Weyl increment of key word 0 (golden ratio) */
#define PHILOX_W1 0xBB67AE85u /* Weyl increment of key word 1 (sqrt(3) - 1) */

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { /* the key schedule advances between rounds */
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Stream addressing.  reading: block q of stream (seed, domain) is Philox
 * with counter (lo32 q, hi32 q, domain, 0) and key (lo32 seed, hi32 seed).
 * Domains: 0 perturbation noise, 3 partition permutation. */
void orc_block(uint64_t seed, uint32_t domain, uint64_t q, uint32_t out[4])
{
    uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), domain, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    orc_philox4x32_10(ctr, key, out);
}

/* ------------------------------------------------------------------------- */
/* Gaussian noise: eps ~ N(0, I) of Eq. (3) and Eq. (8).                       */
/* reading: Box-Muller on pairs of words.  Word a gives the radius through    */
/* U(a) = ((a >> 8) + 1) * 2^-24 in (0, 1]; word b gives the angle 2*pi*U(b). */
/* ------------------------------------------------------------------------- */

double orc_uniform_open0(uint32_t x)
{
    return (double)((x >> 8) + 1u) * 0x1p-24;
}

/* rho = sqrt(-2 ln U(a)); U(a) = 1 gives exactly 0. */
double orc_bm_radius(uint32_t a)
{
    double u = orc_uniform_open0(a);
    return sqrt(-2.0 * log(u));
}

/* (cos, sin) of the angle 2*pi*U(b).  2*U(b) = m * 2^-23 with m = (b >> 8) + 1
 * in [1, 2^24], so the angle is pi * m * 2^-23 and a full turn is m = 2^24.
 * The quadrant and the remainder come from m exactly (integer arithmetic), so
 * the angles 0, pi/2, pi, 3pi/2 give exact zeros and ones. */
void orc_bm_angle(uint32_t b, double* cos_out, double* sin_out)
{
    uint32_t m = (b >> 8) + 1u;
    uint32_t quadrant = (m >> 22) & 3u;          /* m = 2^24 wraps to quadrant 0 */
    uint32_t rem = m & ((1u << 22) - 1u);        /* angle in quadrant = pi*rem*2^-23 */
    double cr, sr;                               /* cos(pi r), sin(pi r), r = rem*2^-23 in [0, 1/2) */
    if (rem <= (1u << 21)) {                     /* r <= 1/4 */
        double r = (double)rem * 0x1p-23;
        cr = cos(M_PI * r);
        sr = sin(M_PI * r);
    } else {                                     /* r > 1/4: use t = 1/2 - r, exact */
        double t = (double)((1u << 22) - rem) * 0x1p-23;
        cr = sin(M_PI * t);
        sr = cos(M_PI * t);
    }
    switch (quadrant) {
    case 0: *cos_out = cr;  *sin_out = sr;  break;
    case 1: *cos_out = -sr; *sin_out = cr;  break;
    case 2: *cos_out = -cr; *sin_out = -sr; break;
    default: *cos_out = sr; *sin_out = -cr; break;
    }
}

/* Vector forms of the two halves of the transform, for exhaustive checks. */
void orc_bm_radius_many(const uint32_t* a, int64_t n, double* out)
{
    int64_t k;
#pragma omp parallel for schedule(static)
    for (k = 0; k < n; ++k)
        out[k] = orc_bm_radius(a[k]);
}

void orc_bm_angle_many(const uint32_t* b, int64_t n, double* cos_out, double* sin_out)
{
    int64_t k;
#pragma omp parallel for schedule(static)
    for (k = 0; k < n; ++k)
        orc_bm_angle(b[k], &cos_out[k], &sin_out[k]);
}

/* Noise value for position j of the stream of `seed`: block q = j / 4 gives
 * four normals; positions 4q, 4q+1 use words (x0, x1) and 4q+2, 4q+3 use
 * (x2, x3); the even position takes the cosine, the odd one the sine.  The
 * double product is rounded once to fp32. */
float orc_normal(uint64_t seed, int64_t j)
{
    return orc_normal_domain(seed, ORC_DOMAIN_NOISE, j);
}

/* The same transform on the words of another stream domain (domain 1:
 * synthetic weight initialisation). */
float orc_normal_domain(uint64_t seed, uint32_t domain, int64_t j)
{
    uint32_t x[4];
    orc_block(seed, domain, (uint64_t)j >> 2, x);
    int t = (int)(j & 3);
    uint32_t a = (t < 2) ? x[0] : x[2];
    uint32_t b = (t < 2) ? x[1] : x[3];
    double rho = orc_bm_radius(a);
    double c, s;
    orc_bm_angle(b, &c, &s);
    return (float)(rho * ((t & 1) ? s : c));
}

void orc_blocks(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks, uint32_t* out)
{
    int64_t b;
#pragma omp parallel for schedule(static)
    for (b = 0; b < nblocks; ++b)
        orc_block(seed, domain, q0 + (uint64_t)b, out + 4 * b);
}

void orc_normals(uint64_t seed, int64_t j0, int64_t n, float* out)
{
    int64_t k;
#pragma omp parallel for schedule(static)
    for (k = 0; k < n; ++k)
        out[k] = orc_normal(seed, j0 + k);
}

/* Seeded normal fill: w[j] = cast(stddev * z_j) with z_j the normal of
 * position j in stream (seed, domain); the product is one fp32 multiply,
 * then bf16 rounding for bf16 storage. */
int orc_fill_normal(void* w, int dtype, int64_t n, uint64_t seed, uint32_t domain, float stddev)
{
    int64_t j;
    if (n < 0 || (dtype != ORC_BF16 && dtype != ORC_F32)) return -1;
#pragma omp parallel for schedule(static)
    for (j = 0; j < n; ++j) {
        float v = stddev * orc_normal_domain(seed, domain, j);
        if (dtype == ORC_BF16)
            ((uint16_t*)w)[j] = orc_f32_to_bf16(v);
        else
            ((float*)w)[j] = v;
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* bf16 storage: round to nearest even from fp32; a NaN stays a quiet NaN.    */
/* ------------------------------------------------------------------------- */

uint16_t orc_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

float orc_bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static float load_w(const void* w, int dtype, int64_t i)
{
    if (dtype == ORC_BF16)
        return orc_bf16_to_f32(((const uint16_t*)w)[i]);
    return ((const float*)w)[i];
}

static void store_w(void* w, int dtype, int64_t i, float x)
{
    if (dtype == ORC_BF16)
        ((uint16_t*)w)[i] = orc_f32_to_bf16(x);
    else
        ((float*)w)[i] = x;
}

/* Position j of a subspace lives at parameter index offset + j (contiguous) or
 * index[offset + j] (an index map), as the embedding P_k of Eq. (8). */
static int64_t param_index(const int64_t* index, int64_t offset, int64_t j)
{
    return index ? index[offset + j] : offset + j;
}

/* ------------------------------------------------------------------------- */
/* Perturbation, Eq. (8) and Alg. 1: theta_{k,i} = theta + sigma_k P_k eps.    */
/* Only the subspace changes.  `sigma` is the effective scale sigma_k of       */
/* Eq. (11); `sign` (+1 or -1) allows mirrored pairs.  j0 is the position of   */
/* element 0 of the call within the subspace, so a window of a large subspace  */
/* can be evaluated on its own.                                                */
/* aux_mode SNAPSHOT: snap[j] receives the pre-perturbation value (the weight  */
/*   backup of Sec. 3.3 / Supp. A.8, "CPU Weight Backup").                     */
/* aux_mode MASTER: the source value is the fp32 master[j] instead of w.       */
/* aux_mode BACKUP: w is first restored from an existing backup aux[j] (dtype  */
/*   of w), then perturbed: one backup of the pre-update weights serves every  */
/*   member of a step.                                                         */
/* ------------------------------------------------------------------------- */

int orc_perturb(void* w, int dtype, int64_t offset, int64_t length, const int64_t* index,
                int64_t j0, float sigma, uint64_t seed, int sign, void* aux, int aux_mode)
{
    if (sign != 1 && sign != -1) return ORC_ERR;
    if (aux_mode == ORC_AUX_BACKUP) {
        if (orc_restore(w, dtype, offset, length, index, j0, sigma, seed, sign, aux, ORC_AUX_SNAPSHOT) != ORC_OK)
            return ORC_ERR;
        return orc_perturb(w, dtype, offset, length, index, j0, sigma, seed, sign, NULL, ORC_AUX_NONE);
    }
    float scale = (float)sign * sigma; /* exact: a sign flip */
    int64_t j;
#pragma omp parallel for schedule(static)
    for (j = 0; j < length; ++j) {
        int64_t i = param_index(index, offset, j);
        float base;
        if (aux_mode == ORC_AUX_MASTER) {
            base = ((const float*)aux)[j];
        } else {
            base = load_w(w, dtype, i);
            if (aux_mode == ORC_AUX_SNAPSHOT) {
                if (dtype == ORC_BF16)
                    ((uint16_t*)aux)[j] = ((const uint16_t*)w)[i];
                else
                    ((float*)aux)[j] = ((const float*)w)[i];
            }
        }
        float z = orc_normal(seed, j0 + j);
        store_w(w, dtype, i, fmaf(scale, z, base));
    }
    return ORC_OK;
}

/* Restore.  SNAPSHOT and MASTER copy the backup back (exact, the reason the
 * paper keeps a backup instead of subtracting, Sec. 3.3).  NONE subtracts the
 * replayed perturbation, which is not an identity in floating point. */
int orc_restore(void* w, int dtype, int64_t offset, int64_t length, const int64_t* index,
                int64_t j0, float sigma, uint64_t seed, int sign, const void* aux, int aux_mode)
{
    if (sign != 1 && sign != -1) return ORC_ERR;
    float scale = -(float)sign * sigma;
    int64_t j;
#pragma omp parallel for schedule(static)
    for (j = 0; j < length; ++j) {
        int64_t i = param_index(index, offset, j);
        if (aux_mode == ORC_AUX_SNAPSHOT) {
            if (dtype == ORC_BF16)
                ((uint16_t*)w)[i] = ((const uint16_t*)aux)[j];
            else
                ((float*)w)[i] = ((const float*)aux)[j];
        } else if (aux_mode == ORC_AUX_MASTER) {
            store_w(w, dtype, i, ((const float*)aux)[j]);
        } else {
            float z = orc_normal(seed, j0 + j);
            store_w(w, dtype, i, fmaf(scale, z, load_w(w, dtype, i)));
        }
    }
    return ORC_OK;
}

/* Master staging: master[j] = fp32 value of the subspace's weight (exact). */
int orc_stage_master(const void* w, int dtype, int64_t offset, int64_t length,
                     const int64_t* index, float* master)
{
    int64_t j;
#pragma omp parallel for schedule(static)
    for (j = 0; j < length; ++j)
        master[j] = load_w(w, dtype, param_index(index, offset, j));
    return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Reward normalisation.                                                       */
/* Z: Eq. (5) / Eq. (12): mean and population standard deviation (divide by    */
/*    the count), then (r - mu) / s.  reading: s = 0 (all rewards equal) gives */
/*    0 for every member, i.e. no update.                                      */
/* RANK: reading: centred average rank a / (n - 1) - 1/2, where a is the       */
/*    0-based rank and ties share the mean of their ranks; n = 1 gives 0.      */
/* group == NULL standardises all rewards jointly (Eq. 12); otherwise each     */
/* group separately (the independent-standardisation ablation, Sec. 4.4).      */
/* A non-finite reward zeroes every output and returns status 1.              */
/* ------------------------------------------------------------------------- */

int orc_normalize(const float* r, int n, int mode, const int* group, float* out, int* status)
{
    *status = 0;
    for (int i = 0; i < n; ++i) {
        if (!isfinite(r[i])) {
            for (int k = 0; k < n; ++k) out[k] = 0.0f;
            *status = 1;
            return ORC_OK;
        }
    }
    for (int i = 0; i < n; ++i) {
        int gi = group ? group[i] : 0;
        int count = 0;
        for (int j = 0; j < n; ++j)
            if ((group ? group[j] : 0) == gi) ++count;
        if (mode == ORC_NORM_Z) {
            double sum = 0.0;
            for (int j = 0; j < n; ++j)
                if ((group ? group[j] : 0) == gi) sum += (double)r[j];
            double mu = sum / (double)count;
            double ss = 0.0;
            for (int j = 0; j < n; ++j)
                if ((group ? group[j] : 0) == gi) {
                    double dev = (double)r[j] - mu;
                    ss += dev * dev;
                }
            double s = sqrt(ss / (double)count);
            out[i] = (s > 0.0) ? (float)(((double)r[i] - mu) / s) : 0.0f;
        } else {
            int less = 0, equal = 0;
            for (int j = 0; j < n; ++j) {
                if ((group ? group[j] : 0) != gi) continue;
                if (r[j] < r[i]) ++less;
                else if (r[j] == r[i]) ++equal;
            }
            if (count == 1) {
                out[i] = 0.0f;
            } else {
                double a = (double)less + 0.5 * (double)(equal - 1);
                out[i] = (float)(a / (double)(count - 1) - 0.5);
            }
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* ES update, Eq. (6) and Eq. (13), with seed replay (Sec. 3.3).               */
/*   theta_S += step * sum_i rhat_i * eps_i                                    */
/* step = alpha / (n * sigma)  (scale_mode 0, the OpenAI-ES form) or           */
/* step = alpha / n            (scale_mode 1, Eq. 6 / Eq. 13 with n = N_k).    */
/* Members that share a seed share a noise vector (mirrored pairs); their     */
/* coefficients are summed first: c_u = sum over members with seed u of       */
/* sign * rhat.  Everything is accumulated in double in the order of first    */
/* appearance of each seed.                                                    */
/* master != NULL: master[j] is updated and the weight becomes its rounding.  */
/* ------------------------------------------------------------------------- */

int orc_update(void* w, int dtype, int64_t offset, int64_t length, const int64_t* index,
               int64_t j0, float* master, int n, const uint64_t* seeds, const int8_t* signs,
               const float* rnorm, float alpha, float sigma, int scale_mode)
{
    if (n < 1) return ORC_ERR;
    uint64_t* useed = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
    double* coef = (double*)malloc(sizeof(double) * (size_t)n);
    if (!useed || !coef) { free(useed); free(coef); return ORC_ERR; }
    int nu = 0;
    for (int i = 0; i < n; ++i) {
        if (signs[i] != 1 && signs[i] != -1) { free(useed); free(coef); return ORC_ERR; }
        int u = 0;
        while (u < nu && useed[u] != seeds[i]) ++u;
        if (u == nu) { useed[nu] = seeds[i]; coef[nu] = 0.0; ++nu; }
        coef[u] += (double)signs[i] * (double)rnorm[i];
    }
    double step = (scale_mode == ORC_SCALE_ALPHA_OVER_N_SIGMA)
                      ? (double)alpha / ((double)n * (double)sigma)
                      : (double)alpha / (double)n;
    int64_t j;
#pragma omp parallel for schedule(static)
    for (j = 0; j < length; ++j) {
        double acc = 0.0;
        for (int u = 0; u < nu; ++u)
            acc += coef[u] * (double)orc_normal(useed[u], j0 + j);
        int64_t i = param_index(index, offset, j);
        if (master) {
            float m = (float)((double)master[j] + step * acc);
            master[j] = m;
            store_w(w, dtype, i, m);
        } else {
            float x = (float)((double)load_w(w, dtype, i) + step * acc);
            store_w(w, dtype, i, x);
        }
    }
    free(useed);
    free(coef);
    return ORC_OK;
}

/* One CoPES step's update, Eq. (13) and the last loop of Alg. 1:            */
/*   g_k = (1/N_k) sum_i rhat_{k,i} eps_{k,i};  theta+ = theta + alpha sum_k P_k g_k */
/* (with step_k = alpha / (N_k sigma_k) under scale_mode 0).  Subspace k is    */
/* positions [offsets[k], offsets[k+1]) of the parameters or of `index`; its  */
/* members are those with subspace[i] == k, in order.  Supports are disjoint, */
/* so the subspaces are updated one after the other from the same theta.     */
int orc_update_step(void* w, int dtype, int K, const int64_t* offsets, const int64_t* index, int n,
                    const uint64_t* seeds, const int8_t* signs, const int* subspace, const float* rnorm,
                    float alpha, const float* sigmas, int scale_mode)
{
    uint64_t* ks = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
    int8_t* kg = (int8_t*)malloc((size_t)n);
    float* kr = (float*)malloc(sizeof(float) * (size_t)n);
    if (!ks || !kg || !kr) { free(ks); free(kg); free(kr); return ORC_ERR; }
    int rc = ORC_OK;
    for (int k = 0; k < K && rc == ORC_OK; ++k) {
        int nk = 0;
        for (int i = 0; i < n; ++i)
            if (subspace[i] == k) { ks[nk] = seeds[i]; kg[nk] = signs[i]; kr[nk] = rnorm[i]; ++nk; }
        if (nk == 0) continue;
        rc = orc_update(w, dtype, offsets[k], offsets[k + 1] - offsets[k], index, 0, NULL, nk, ks, kg, kr,
                        alpha, sigmas[k], scale_mode);
    }
    free(ks); free(kg); free(kr);
    return rc;
}

/* ------------------------------------------------------------------------- */
/* Partition of Eq. (7): disjoint subspaces covering all d indices, sizes     */
/* d/K (within one when K does not divide d).                                  */
/* CONTIGUOUS: offsets given by the caller (checked monotone from 0 to d) or  */
/*   floor(k d / K).                                                            */
/* PERMUTATION: reading: a keyed pseudo-random permutation E of [0, d) is a    */
/*   balanced Feistel network on b bits (b = max(2, ceil(log2 d)) rounded up   */
/*   to even, h = b/2; eight rounds (L, R) <- (R, L xor F_r(R)), with          */
/*   F_r(R) = word 0 of Philox block (seed, domain 3, q = r * 2^32 + R), masked */
/*   to h bits), restricted to [0, d) by cycle-walking (Black and Rogaway,     */
/*   "Ciphers with arbitrary finite domains", CT-RSA 2002).  Element i goes to */
/*   subspace floor(E(i) K / d); each subspace lists its elements ascending.   */
/*   Because E is a bijection, subspace k starts at ceil(k d / K).  Eight      */
/*   rounds rather than four: with four, the partitions of a six-element set   */
/*   are visibly non-uniform over seeds (chi-square p ~ 1e-13).                */
/* The paper resamples the partition each step from a stored seed (Sec. 3.3,  */
/* Supp. A.8 "Partition Replay").                                              */
/* ------------------------------------------------------------------------- */

#define ORC_FEISTEL_ROUNDS 8

static int feistel_bits(int64_t d)
{
    int b = 0;
    while (b < 63 && ((int64_t)1 << b) < d) ++b; /* ceil(log2 d) */
    if (b < 2) b = 2;
    if (b & 1) ++b;
    return b;
}

static uint64_t feistel_once(uint64_t seed, int h, uint64_t x)
{
    uint64_t mask = ((uint64_t)1 << h) - 1u;
    uint64_t L = x >> h, R = x & mask;
    for (uint64_t r = 0; r < ORC_FEISTEL_ROUNDS; ++r) {
        uint32_t y[4];
        orc_block(seed, ORC_DOMAIN_PARTITION, (r << 32) | R, y);
        uint64_t nl = R;
        uint64_t nr = L ^ ((uint64_t)y[0] & mask);
        L = nl;
        R = nr;
    }
    return (L << h) | R;
}

int64_t orc_prp(uint64_t seed, int64_t d, int64_t x)
{
    int h = feistel_bits(d) / 2;
    uint64_t y = feistel_once(seed, h, (uint64_t)x);
    while (y >= (uint64_t)d)
        y = feistel_once(seed, h, y);
    return (int64_t)y;
}

int32_t orc_bucket(uint64_t seed, int64_t d, int32_t K, int64_t i)
{
    unsigned __int128 e = (unsigned __int128)(uint64_t)orc_prp(seed, d, i);
    return (int32_t)((e * (unsigned __int128)(uint32_t)K) / (unsigned __int128)(uint64_t)d);
}

int orc_partition(int mode, int64_t d, int32_t K, uint64_t seed, const int64_t* bounds,
                  int64_t* offsets, int64_t* index)
{
    if (d < 1 || K < 1 || (int64_t)K > d) return ORC_ERR;
    if (mode == ORC_PART_CONTIGUOUS) {
        if (bounds) {
            if (bounds[0] != 0 || bounds[K] != d) return ORC_ERR;
            for (int k = 0; k < K; ++k)
                if (bounds[k + 1] < bounds[k]) return ORC_ERR;
            for (int k = 0; k <= K; ++k) offsets[k] = bounds[k];
        } else {
            for (int k = 0; k <= K; ++k)
                offsets[k] = (int64_t)(((unsigned __int128)(uint64_t)d * (uint64_t)k) / (uint64_t)K);
        }
        return ORC_OK;
    }
    if (mode != ORC_PART_PERMUTATION) return ORC_ERR;
    for (int k = 0; k <= K; ++k) /* ceil(k d / K) */
        offsets[k] = (int64_t)(((unsigned __int128)(uint64_t)d * (uint64_t)k + (uint64_t)K - 1u) / (uint64_t)K);
    if (!index) return ORC_OK;
    int32_t* bucket = (int32_t*)malloc(sizeof(int32_t) * (size_t)d);
    int64_t* fill = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
    if (!bucket || !fill) { free(bucket); free(fill); return ORC_ERR; }
    int64_t i;
#pragma omp parallel for schedule(static)
    for (i = 0; i < d; ++i)
        bucket[i] = orc_bucket(seed, d, K, i);
    for (int k = 0; k < K; ++k) fill[k] = offsets[k];
    for (i = 0; i < d; ++i) /* ascending i keeps every list sorted */
        index[fill[bucket[i]]++] = i;
    int ok = 1;
    for (int k = 0; k < K; ++k)
        if (fill[k] != offsets[k + 1]) ok = 0;
    free(bucket);
    free(fill);
    return ok ? ORC_OK : ORC_ERR;
}

/* Chunk-granular partition (Sec. 3.3; Supp. A.8 "Partition Replay"): the d
 * parameters form ceil(d / chunk) chunks of `chunk` consecutive parameters
 * (the last may be shorter), and the chunk ids are partitioned exactly as
 * elements are above.  lengths[k] is the number of parameters in the chunks
 * of subspace k. */
int orc_partition_chunks(int64_t d, int64_t chunk, int32_t K, uint64_t seed, int64_t* list_offsets,
                         int64_t* lengths, int64_t* chunks)
{
    if (d < 1 || chunk < 1) return ORC_ERR;
    int64_t n_chunks = (d + chunk - 1) / chunk;
    int rc = orc_partition(ORC_PART_PERMUTATION, n_chunks, K, seed, NULL, list_offsets, chunks);
    if (rc != ORC_OK) return rc;
    for (int k = 0; k < K; ++k) {
        int64_t total = 0;
        for (int64_t t = list_offsets[k]; t < list_offsets[k + 1]; ++t) {
            int64_t first = chunks[t] * chunk;
            int64_t last = first + chunk < d ? first + chunk : d;
            total += last - first;
        }
        lengths[k] = total;
    }
    return ORC_OK;
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
