/*
 * cpes_oracle.h -- declarations of the CPU oracle (test infrastructure only).
 * Host pointers throughout; bf16 buffers are arrays of uint16_t bit patterns.
 * The enum values equal the GPU library's by convention (the tests pass the
 * same integers to both), but neither side includes the other's header.
 */
#ifndef CPES_ORACLE_H
#define CPES_ORACLE_H

#include <stdint.h>

#define ORC_OK 0
#define ORC_ERR (-1)

#define ORC_BF16 0
#define ORC_F32 1

#define ORC_AUX_NONE 0
#define ORC_AUX_SNAPSHOT 1
#define ORC_AUX_MASTER 2
#define ORC_AUX_BACKUP 3

#define ORC_NORM_Z 0
#define ORC_NORM_RANK 1

#define ORC_SCALE_ALPHA_OVER_N_SIGMA 0
#define ORC_SCALE_ALPHA_OVER_N 1

#define ORC_PART_CONTIGUOUS 0
#define ORC_PART_PERMUTATION 1

#define ORC_DOMAIN_NOISE 0u
#define ORC_DOMAIN_PARTITION 3u

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
void orc_block(uint64_t seed, uint32_t domain, uint64_t q, uint32_t out[4]);
double orc_uniform_open0(uint32_t x);
double orc_bm_radius(uint32_t a);
void orc_bm_angle(uint32_t b, double* cos_out, double* sin_out);
void orc_bm_radius_many(const uint32_t* a, int64_t n, double* out);
void orc_bm_angle_many(const uint32_t* b, int64_t n, double* cos_out, double* sin_out);
void orc_blocks(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks, uint32_t* out);
float orc_normal(uint64_t seed, int64_t j);
float orc_normal_domain(uint64_t seed, uint32_t domain, int64_t j);
int orc_fill_normal(void* w, int dtype, int64_t n, uint64_t seed, uint32_t domain, float stddev);
void orc_normals(uint64_t seed, int64_t j0, int64_t n, float* out);
uint16_t orc_f32_to_bf16(float f);
float orc_bf16_to_f32(uint16_t h);

int orc_perturb(void* w, int dtype, int64_t offset, int64_t length, const int64_t* index,
                int64_t j0, float sigma, uint64_t seed, int sign, void* aux, int aux_mode);
int orc_restore(void* w, int dtype, int64_t offset, int64_t length, const int64_t* index,
                int64_t j0, float sigma, uint64_t seed, int sign, const void* aux, int aux_mode);
int orc_stage_master(const void* w, int dtype, int64_t offset, int64_t length,
                     const int64_t* index, float* master);
int orc_normalize(const float* r, int n, int mode, const int* group, float* out, int* status);
int orc_update(void* w, int dtype, int64_t offset, int64_t length, const int64_t* index,
               int64_t j0, float* master, int n, const uint64_t* seeds, const int8_t* signs,
               const float* rnorm, float alpha, float sigma, int scale_mode);

int orc_update_step(void* w, int dtype, int K, const int64_t* offsets, const int64_t* index, int n,
                    const uint64_t* seeds, const int8_t* signs, const int* subspace, const float* rnorm,
                    float alpha, const float* sigmas, int scale_mode);

int64_t orc_prp(uint64_t seed, int64_t d, int64_t x);
int32_t orc_bucket(uint64_t seed, int64_t d, int32_t K, int64_t i);
int orc_partition(int mode, int64_t d, int32_t K, uint64_t seed, const int64_t* bounds,
                  int64_t* offsets, int64_t* index);
int orc_partition_chunks(int64_t d, int64_t chunk, int32_t K, uint64_t seed, int64_t* list_offsets,
                         int64_t* lengths, int64_t* chunks);
int orc_num_threads(void);

#endif
