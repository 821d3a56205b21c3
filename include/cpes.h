/*
 * cpes.h -- C ABI of the CoPES parameter-space hot path for AMD Instinct
 * MI355X (gfx950).
 *
 * CoPES ("Cooperative Coevolution for Resource-Constrained Agentic LLM
 * Post-Training", arXiv 2608.02391) is an evolution strategy over all
 * parameters of a model.  One step (Alg. 1) partitions the d parameters into K
 * disjoint subspaces (Eq. 7), evaluates seed-defined Gaussian perturbations of
 * one subspace at a time (Eq. 8, scale sigma_k of Eq. 11), standardises the
 * rewards of all members jointly (Eq. 12) and adds the reward-weighted noise
 * back to the parameters (Eq. 13; Eq. 6 for standard ES).  Noise is never
 * stored: every call regenerates it from the member's seed (Sec. 3.3 and
 * Supp. A.8, "Seed Replay and Chunking"), and the pre-perturbation weights are
 * restored from a backup rather than by subtraction ("CPU Weight Backup").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers named *_dev are device pointers (e.g. a torch tensor's data_ptr());
 * pointers named *_host are host pointers.  The caller owns every buffer; the
 * library keeps no pointer and no state between calls besides a thread-local
 * error string.  `stream` is a hipStream_t passed as void* (NULL = the null
 * stream).  Every call only enqueues work on `stream` and returns without
 * synchronising; a kernel failure surfaces at the caller's next
 * synchronisation.  Arguments are validated on the host before anything is
 * enqueued, so a call that returns an error has had no effect.  No call
 * allocates device memory; scratch space comes in through `workspace`.
 * Results depend only on the arguments (not on the stream, launch geometry or
 * run).
 *
 * Weights are a flat buffer of `numel` elements of dtype CPES_BF16 or
 * CPES_F32.  A subspace (cpes_subspace) lists `length` positions j = 0 ..
 * length-1 -- the embedding P_k of Eq. 8.  Position j is parameter
 *   offset + j                                  (index == NULL),
 *   index[offset + j]                           (index != NULL, chunk == 0), or
 *   index[offset + j / chunk] * chunk + j % chunk
 *                                               (index != NULL, chunk > 0:
 *                                                the map names chunks of `chunk`
 *                                                consecutive parameters),
 * index being a device array of int64; an element map may instead be a
 * uint32 array (index32, models of at most 2^32 parameters).  Entries that
 * would address outside [0, numel) are skipped.
 *
 * Noise.  Position j of a subspace draws noise index i = noise_offset + j
 * (noise_offset = 0 for a whole subspace; a shard of one passes its start).
 * Noise index i of a member with seed s is
 *   eps_i = BoxMuller(Philox4x32-10(counter = (lo32 q, hi32 q, 0, 0),
 *                                   key = (lo32 s, hi32 s)), i mod 4),
 * q = i / 4: words (x0, x1) give indices 4q and 4q+1, words (x2, x3) give
 * 4q+2 and 4q+3; radius sqrt(-2 ln U(a)), angle 2 pi U(b), U(x) = ((x >> 8) +
 * 1) 2^-24; cosine for the even index, sine for the odd one; evaluated in
 * fp64 and rounded once to fp32.
 */
#ifndef CPES_H
#define CPES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CPES_ABI_VERSION 8

/* Exported symbols (the library is built with hidden default visibility). */
#define CPES_API __attribute__((visibility("default")))

/* Status codes returned by every int-valued entry point. */
enum cpes_status {
    CPES_OK = 0,
    CPES_ERR_INVALID_ARGUMENT = -1, /* a null, out-of-range or inconsistent argument */
    CPES_ERR_UNSUPPORTED = -2,      /* valid but beyond the library's limits (see each call) */
    CPES_ERR_WORKSPACE = -3,        /* workspace missing or smaller than required */
    CPES_ERR_HIP = -4,              /* the HIP runtime reported an error while enqueueing */
};

enum cpes_dtype { CPES_BF16 = 0, CPES_F32 = 1 };
enum cpes_partition_mode { CPES_PART_CONTIGUOUS = 0, CPES_PART_PERMUTATION = 1 };
enum cpes_aux_mode { CPES_AUX_NONE = 0, CPES_AUX_SNAPSHOT = 1, CPES_AUX_MASTER = 2, CPES_AUX_BACKUP = 3 };
enum cpes_norm_mode { CPES_NORM_Z = 0, CPES_NORM_RANK = 1 };
enum cpes_scale_mode { CPES_SCALE_ALPHA_OVER_N_SIGMA = 0, CPES_SCALE_ALPHA_OVER_N = 1 };

/* Limits of the library. */
#define CPES_MAX_MEMBERS 256         /* members per cpes_update call */
#define CPES_MAX_REWARDS 4096        /* rewards per cpes_normalize_rewards call */
#define CPES_MAX_GROUPS 1024         /* reward groups per cpes_normalize_rewards call */
#define CPES_MAX_PERMUTATION_K 256   /* subspaces of a CPES_PART_PERMUTATION partition */
#define CPES_MAX_STEP_SUBSPACES 32   /* subspaces per cpes_update_step call */
#define CPES_STATIC_MAX_CHUNKS (1 << 20) /* chunks per cpes_partition_chunks_static call */

typedef struct cpes_subspace {
    int64_t offset;          /* first parameter (no map) or first map entry */
    int64_t length;          /* number of positions d_k, >= 0 */
    const int64_t* index;    /* NULL, or device int64 map (parameters or chunk ids) */
    int64_t chunk;           /* 0, or a power of two >= 8: index entries name chunks of this size */
    const uint32_t* index32; /* NULL, or device uint32 map of parameters (half the map traffic
                                of `index`; models of at most 2^32 parameters); at most one of
                                index / index32, and chunk = 0 with index32 */
    int64_t noise_offset;    /* 0, or a multiple of 8: position j draws noise index
                                noise_offset + j.  A shard [a, b) of a subspace is
                                {offset + a (or the map entry a), b - a, ..., noise_offset = a}
                                and gets exactly the noise, and the results, of those positions
                                of the whole subspace (a sharded update across GPUs). */
    int64_t flags;           /* 0, or CPES_SUB_ASCENDING (below) */
} cpes_subspace;

/* cpes_subspace.flags.  CPES_SUB_ASCENDING: the element map (index or
 * index32) is strictly ascending over the subspace's positions, as the maps
 * of cpes_partition and cpes_partition32 are.  With bf16 weights the
 * perturbations (cpes_perturb, every aux mode) and the restores (cpes_restore
 * from a backup or a master, cpes_restore_from_host) may then read and write
 * whole 128-byte lines of the weights around the subspace's entries (once
 * each), writing the other parameters of those lines back with the values
 * just read, instead of storing the entries one by one: on a dense subspace
 * almost every line is then written in full rather than partially.  Results
 * are those of the entry-by-entry path, provided nothing else writes the same
 * weights while the call runs; with a map that is not strictly ascending they
 * are undefined (every access stays within w, the map and the side buffer).
 * Ignored for other calls, contiguous and chunked subspaces and fp32
 * weights. */
#define CPES_SUB_ASCENDING 1

/*
 * cpes_partition -- subspaces of Eq. (7): disjoint, covering all d indices,
 * sizes d/K (differing by at most one when K does not divide d).  The paper
 * resamples the partition every step from a stored seed and replays it
 * (Sec. 3.3, Supp. A.8 "Partition Replay").
 *
 * mode CPES_PART_CONTIGUOUS: offsets_host[k] = bounds_host[k] (K+1 values,
 *   non-decreasing from 0 to d) or, with bounds_host == NULL, floor(k d / K).
 *   Subspace k is the parameter range [offsets[k], offsets[k+1]).  Host only:
 *   nothing is enqueued, index_dev / workspace may be NULL.
 * mode CPES_PART_PERMUTATION: element i belongs to subspace
 *   floor(E(i) K / d), where E is a keyed pseudo-random permutation of [0, d):
 *   an 8-round balanced Feistel network on b = max(2, ceil(log2 d)) (rounded
 *   up to even) bits whose round r function is word 0 of the Philox block
 *   (counter (R, r, 3, 0), key seed) masked to b/2 bits, restricted to [0, d)
 *   by cycle-walking.  index_dev (device int64[d]) receives, for each k, the
 *   members of subspace k in ascending order at [offsets[k], offsets[k+1]),
 *   and offsets_host[k] = ceil(k d / K) (exact because E is a bijection).
 *   Requires 1 <= K <= CPES_MAX_PERMUTATION_K, d < 2^55 and a device workspace of
 *   cpes_partition_workspace_bytes() bytes (16-byte aligned).
 * status_dev: NULL, or a device int32 set to 0, or to 1 if a cycle walk
 *   exceeded its bound (cannot happen for a bijection; a safety net).
 * Errors: d < 1 or d >= 2^62, K < 1 or K > d, bad bounds, mode unknown,
 *   index_dev NULL for PERMUTATION -> CPES_ERR_INVALID_ARGUMENT; K above the
 *   limit -> CPES_ERR_UNSUPPORTED; workspace too small -> CPES_ERR_WORKSPACE.
 */
CPES_API int cpes_partition(int mode, int64_t d, int32_t K, uint64_t seed, const int64_t* bounds_host,
                   int64_t* offsets_host, int64_t* index_dev, void* workspace_dev,
                   size_t workspace_bytes, int32_t* status_dev, void* stream);

/*
 * cpes_partition32 -- the CPES_PART_PERMUTATION partition of cpes_partition
 * written as a uint32 map (index_dev: device uint32[d]) for d <= 2^32: half
 * the memory and half the map traffic of the int64 map, same entries.  Use it
 * through cpes_subspace.index32.  Workspace as
 * cpes_partition_workspace_bytes(CPES_PART_PERMUTATION, d, K).
 * Errors: d < 1 or d > 2^32, K < 1 or K > d, null pointers ->
 *   CPES_ERR_INVALID_ARGUMENT; otherwise as cpes_partition.
 */
CPES_API int cpes_partition32(int64_t d, int32_t K, uint64_t seed, int64_t* offsets_host, uint32_t* index_dev,
                     void* workspace_dev, size_t workspace_bytes, int32_t* status_dev, void* stream);

/* Workspace bytes cpes_partition needs (0 for CONTIGUOUS); 0 for invalid arguments. */
CPES_API size_t cpes_partition_workspace_bytes(int mode, int64_t d, int32_t K);

/*
 * cpes_partition_chunks -- the chunk-granular random partition the paper runs
 * (Sec. 3.3; Supp. A.8 "Partition Replay": the assignment of chunks to
 * subspaces is replayed from a stored seed).  The d parameters form n_chunks = ceil(d /
 * chunk) chunks of `chunk` consecutive parameters (the last may be shorter);
 * chunk c belongs to subspace floor(E(c) K / n_chunks), E being the keyed
 * permutation of cpes_partition (CPES_PART_PERMUTATION) on [0, n_chunks).
 *   chunks_dev (device int64[n_chunks]) receives the chunk ids of each
 *   subspace, ascending, at [list_offsets[k], list_offsets[k+1]);
 *   list_offsets_host[k] = ceil(k n_chunks / K) (host, K+1);
 *   lengths_host[k] = parameters in subspace k (host, K; they sum to d).
 * Subspace k is then cpes_subspace{list_offsets[k], lengths[k], chunks_dev,
 * chunk}: every 16-byte unit is contiguous, so kernels stream it at full
 * bandwidth.  chunk must be a power of two, 8 <= chunk <= 2^30; 1 <= K <=
 * min(n_chunks, CPES_MAX_PERMUTATION_K); workspace as
 * cpes_partition_chunks_workspace_bytes(); status_dev as cpes_partition.
 */
CPES_API int cpes_partition_chunks(int64_t d, int64_t chunk, int32_t K, uint64_t seed,
                                   int64_t* list_offsets_host, int64_t* lengths_host, int64_t* chunks_dev,
                                   void* workspace_dev, size_t workspace_bytes, int32_t* status_dev,
                                   void* stream);

/*
 * cpes_partition_chunks_static -- cpes_partition_chunks with no workspace
 * argument and no allocation of any kind, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Its scratch space is a file-scope device array of
 * the library (2,621,696 bytes: room for n_chunks <= CPES_STATIC_MAX_CHUNKS
 * and K <= CPES_MAX_PERMUTATION_K), which every GPU the library runs on holds
 * until the process ends.  The first call on a device looks up that device's
 * copy (hipGetSymbolAddress; not a stream operation, so make that first call
 * outside a graph capture).  All calls on one GPU share the array and each
 * leaves its contents behind: calls that overlap in time on one GPU (other
 * streams or threads) race and must be serialised by the caller.  Nothing in
 * it needs to start at zero: every call writes each scratch entry before
 * reading it.
 * Arguments, outputs and results as cpes_partition_chunks (bit-identical).
 * Errors: as cpes_partition_chunks; more than CPES_STATIC_MAX_CHUNKS chunks
 *   -> CPES_ERR_UNSUPPORTED; the address lookup failing -> CPES_ERR_HIP.
 */
CPES_API int cpes_partition_chunks_static(int64_t d, int64_t chunk, int32_t K, uint64_t seed,
                                          int64_t* list_offsets_host, int64_t* lengths_host, int64_t* chunks_dev,
                                          int32_t* status_dev, void* stream);

/* Workspace bytes cpes_partition_chunks needs; 0 for invalid arguments. */
CPES_API size_t cpes_partition_chunks_workspace_bytes(int64_t d, int64_t chunk, int32_t K);

/*
 * cpes_perturb -- theta_{k,i} = theta + sigma_k P_k eps_{k,i} (Eq. 8, Alg. 1),
 * in place on the subspace `s` of w (numel elements of `dtype`):
 *   w[p(j)] = cast(fmaf(sign * sigma, eps_j(seed), src_j)),  j < s->length,
 * one fp32 fused multiply-add, then round-to-nearest-even for bf16.
 * sigma is the effective scale sigma_k = sigma sqrt(d / d_k) (Eq. 11);
 * sign is +1 or -1 (mirrored pairs).
 *   aux_mode CPES_AUX_NONE:     src_j = w[p(j)]; aux ignored.
 *   aux_mode CPES_AUX_SNAPSHOT: src_j = w[p(j)], and aux (device, dtype of w,
 *                               s->length elements) receives aux[j] = w[p(j)]
 *                               before the change: the weight backup.
 *   aux_mode CPES_AUX_MASTER:   src_j = ((const float*)aux)[j], an fp32 master
 *                               of the subspace (CPES_BF16 weights only).
 *   aux_mode CPES_AUX_BACKUP:   src_j = aux[j], an existing backup (dtype of w)
 *                               of the unperturbed subspace, read only; w is
 *                               not read.  Equal to restoring from the backup
 *                               and then perturbing, in one pass.  Every member
 *                               of a step perturbs the same pre-update weights,
 *                               so one backup serves all of them.
 * Parameters outside the subspace keep their values (through a map flagged
 * CPES_SUB_ASCENDING, bf16 lines around the entries are rewritten with the
 * values just read; see cpes_subspace.flags).
 * Errors: w NULL, s NULL, length < 0, contiguous range beyond numel, dtype /
 *   aux_mode unknown, aux NULL when needed, sign not +-1, sigma negative or
 *   not finite, MASTER with fp32 weights -> CPES_ERR_INVALID_ARGUMENT.
 */
CPES_API int cpes_perturb(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float sigma,
                 uint64_t seed, int32_t sign, void* aux_dev, int aux_mode, void* stream);

/*
 * cpes_restore -- undo a perturbation (Sec. 3.3):
 *   CPES_AUX_SNAPSHOT: w[p(j)] = aux[j] (bit copy; exact).
 *   CPES_AUX_MASTER:   w[p(j)] = rne_bf16(((const float*)aux)[j]) (exact when
 *                      the master was staged from w).
 *   CPES_AUX_NONE:     replay: w[p(j)] = cast(fmaf(-sign * sigma, eps_j, w[p(j)])).
 *                      Not an identity in floating point; the paper's reason for
 *                      keeping a backup.  Differs by at most one fp32 ulp (more
 *                      after bf16 rounding).
 * Arguments and errors as cpes_perturb (sigma, seed, sign only used by NONE).
 */
CPES_API int cpes_restore(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float sigma,
                 uint64_t seed, int32_t sign, const void* aux_dev, int aux_mode, void* stream);

/*
 * cpes_backup_to_host -- backup_host[j] = w[p(j)] (bit copy), the weight
 * backup in host memory (Sec. 3.3; Supp. A.8, CPU weight backup): the
 * pre-perturbation weights of the subspace leave the GPU, so the backup adds
 * no device-resident copy.
 * cpes_restore_from_host -- w[p(j)] = backup_host[j] (bit copy), the restore
 * after each perturbed-model evaluation.
 *   backup_host: s->length elements of `dtype`, PINNED host memory the device
 *                can address (hipHostMalloc, or a torch tensor made with
 *                pin_memory=True); owned by the caller, who keeps it alive and
 *                unmodified until the work on `stream` has finished.
 * A contiguous subspace moves as one DMA copy on `stream`; an index-map or
 * chunked subspace is gathered / scattered by a kernel that reads or writes
 * the pinned buffer over the host link.  Both are asynchronous on `stream`.
 * Errors: as cpes_perturb for w and s; backup_host NULL or not pinned host
 *   memory (pageable, or device memory) -> CPES_ERR_INVALID_ARGUMENT.
 */
CPES_API int cpes_backup_to_host(const void* w_dev, int64_t numel, int dtype, const cpes_subspace* s,
                        void* backup_host, void* stream);
CPES_API int cpes_restore_from_host(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s,
                           const void* backup_host, void* stream);

/*
 * cpes_backup -- backup_dev[j] = w[p(j)] (bit copy), the weight backup of
 * Sec. 3.3 taken on its own, in device memory: for a subspace whose members
 * are perturbed from another source (an fp32 master) but restored from a copy
 * of the weights.  (A member's perturbation can also take the backup itself:
 * cpes_perturb with CPES_AUX_SNAPSHOT.)
 *   backup_dev: s->length elements of `dtype` in device memory, caller-owned;
 *               it must not overlap w.
 * Errors: as cpes_perturb for w and s; backup_dev NULL -> CPES_ERR_INVALID_ARGUMENT.
 */
CPES_API int cpes_backup(const void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, void* backup_dev,
                void* stream);

/*
 * cpes_stage_master -- master_dev[j] = fp32 value of w[p(j)] (exact), the fp32
 * master copy of the active subspace kept while its bf16 weights are
 * perturbed and updated.  Errors as cpes_perturb.
 */
CPES_API int cpes_stage_master(const void* w_dev, int64_t numel, int dtype, const cpes_subspace* s,
                      float* master_dev, void* stream);

/*
 * cpes_normalize_rewards -- reward standardisation.
 *   CPES_NORM_Z:    Eq. (5) / Eq. (12): mu = sum r / n, s = sqrt(sum (r - mu)^2 / n)
 *                   (population std, sums in fp64 in index order);
 *                   out = (r - mu) / s, or 0 for every member when s == 0.
 *   CPES_NORM_RANK: centred average rank a / (n - 1) - 1/2 with a the 0-based
 *                   rank and ties sharing the mean of their ranks; 0 when n == 1.
 * group_dev == NULL standardises all n rewards jointly (Eq. 12).  Otherwise
 * group_dev (device int32[n], values in [0, n_groups)) standardises each group
 * on its own (independent standardisation, the ablation of Sec. 4.4).
 * r_dev and out_dev are device float32[n] and may alias.  status_dev (NULL or
 * device int32) receives 0, 1 if a reward is not finite, or 2 if a group id is
 * out of range; in both failure cases every output is 0 (so an update leaves
 * the weights unchanged).
 * Errors: NULL r_dev / out_dev, n outside [1, CPES_MAX_REWARDS], unknown mode,
 *   n_groups outside [1, n] with group_dev given -> CPES_ERR_INVALID_ARGUMENT;
 *   n_groups above CPES_MAX_GROUPS -> CPES_ERR_UNSUPPORTED.
 */
CPES_API int cpes_normalize_rewards(const float* r_dev, int32_t n, int mode, const int32_t* group_dev,
                           int32_t n_groups, float* out_dev, int32_t* status_dev, void* stream);

/*
 * cpes_update -- seed-replayed ES update of one subspace (Eq. 6 / Eq. 13;
 * Sec. 3.3):  theta_S += step * sum_i sign_i * rnorm_i * eps(seed_i),
 *   step = alpha / (n * sigma)   (CPES_SCALE_ALPHA_OVER_N_SIGMA, OpenAI-ES form)
 *   step = alpha / n             (CPES_SCALE_ALPHA_OVER_N, the paper's form with
 *                                 n = N_k members of this subspace).
 * seeds_host / signs_host (host, n entries; signs +-1) describe the members in
 * the order their rewards appear in rnorm_dev (device float32[n], typically
 * the output of cpes_normalize_rewards).  Members sharing a seed (mirrored
 * pairs) share one noise vector, which is generated once with coefficient
 * sum(sign * rnorm).  Each weight is read once and written once; the weighted
 * noise sum is accumulated in fp32 in order of first appearance of each seed.
 *   master_dev == NULL: w[p(j)] = cast(fmaf(step, acc_j, w[p(j)])).
 *   master_dev != NULL: master[j] = fmaf(step, acc_j, master[j]) and
 *                       w[p(j)] = cast(master[j]) (device float32[length]).
 * Errors: NULL pointers, n outside [1, CPES_MAX_MEMBERS] (UNSUPPORTED above),
 *   a sign not +-1, alpha or sigma not finite, sigma <= 0 with the
 *   OVER_N_SIGMA scale, dtype / scale_mode unknown, contiguous range beyond
 *   numel -> CPES_ERR_INVALID_ARGUMENT.
 */
CPES_API int cpes_update(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float* master_dev,
                int32_t n, const uint64_t* seeds_host, const int8_t* signs_host,
                const float* rnorm_dev, float alpha, float sigma, int scale_mode, void* stream);

/*
 * cpes_update_step -- the whole CoPES update of one step in one launch
 * (Eq. 13; Alg. 1, after joint standardisation): for every subspace k of a
 * partition,  theta_{S_k} += step_k * sum_{i in members of k} sign_i rnorm_i eps(seed_i),
 *   step_k = alpha / (n_k sigma_k)  (CPES_SCALE_ALPHA_OVER_N_SIGMA) or
 *   step_k = alpha / n_k            (CPES_SCALE_ALPHA_OVER_N; Eq. 13 with n_k = N_k),
 * where n_k counts the members of subspace k.  With K = 1 and alpha / N this
 * is the standard ES update of Eq. 6.  Subspaces are disjoint, so the result
 * equals K cpes_update calls in any order.
 * offsets_host (K+1, non-decreasing): subspace k is positions [offsets[k],
 *   offsets[k+1]) -- parameters themselves (index_dev == NULL; offsets[K] <=
 *   numel) or entries of the int64 device map index_dev (e.g. the output of
 *   cpes_partition; a uint32 map goes to cpes_update_step32).  Noise
 *   position j is counted from offsets[k].
 *   With chunk > 0, index_dev holds chunk ids (cpes_partition_chunks),
 *   subspace k is cpes_subspace{offsets[k], lengths_host[k], index_dev, chunk}
 *   and lengths_host (host, K) is required; otherwise lengths_host is ignored.
 * seeds_host / signs_host / subspace_host (host, n entries): member i has seed,
 *   sign +-1 and the subspace it perturbed; rnorm_dev (device float32[n]) its
 *   standardised reward (joint or per group, cpes_normalize_rewards).
 *   Members of one subspace sharing a seed share one noise stream.
 * sigma_host (host, K): the effective sigma_k each subspace was perturbed with.
 * Subspaces without members are left unchanged.  Each weight is read and
 * written once; accumulation in fp32 as in cpes_update.
 * Errors: NULL pointers, K < 1, n < 1, a sign not +-1, a member's subspace
 *   outside [0, K), decreasing offsets, contiguous range beyond numel, alpha
 *   not finite, sigma_k <= 0 for a subspace with members under the
 *   OVER_N_SIGMA scale -> CPES_ERR_INVALID_ARGUMENT; K above
 *   CPES_MAX_STEP_SUBSPACES or n above CPES_MAX_MEMBERS -> CPES_ERR_UNSUPPORTED.
 */
CPES_API int cpes_update_step(void* w_dev, int64_t numel, int dtype, int32_t K, const int64_t* offsets_host,
                              const int64_t* index_dev, int64_t chunk, const int64_t* lengths_host,
                              int32_t n, const uint64_t* seeds_host,
                              const int8_t* signs_host, const int32_t* subspace_host, const float* rnorm_dev,
                              float alpha, const float* sigma_host, int scale_mode, void* stream);

/*
 * cpes_update_step32 -- cpes_update_step over a uint32 element map
 * (index32_dev, e.g. the output of cpes_partition32; models of at most 2^32
 * parameters): subspace k is entries [offsets[k], offsets[k+1]) of the map.
 * Half the map traffic of the int64 map, same result.  No chunk lists.
 * Arguments and errors otherwise as cpes_update_step; index32_dev NULL ->
 * CPES_ERR_INVALID_ARGUMENT.
 */
CPES_API int cpes_update_step32(void* w_dev, int64_t numel, int dtype, int32_t K, const int64_t* offsets_host,
                                const uint32_t* index32_dev, int32_t n, const uint64_t* seeds_host,
                                const int8_t* signs_host, const int32_t* subspace_host, const float* rnorm_dev,
                                float alpha, const float* sigma_host, int scale_mode, void* stream);

/* ---------------- test hooks and measurement utilities ------------------ */

/* out_dev[4 b + t] = word t of the Philox block q0 + b of stream (seed, domain),
 * b < nblocks.  Errors: out_dev NULL, nblocks < 0. */
CPES_API int cpes_debug_philox(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks,
                      uint32_t* out_dev, void* stream);

/* out_dev[k] = eps_{j0 + k}(seed) for k < n (the noise perturb/update use). */
CPES_API int cpes_debug_normals(uint64_t seed, int64_t j0, int64_t n, float* out_dev, void* stream);

/* The two halves of the normal transform on the grid m = m0 + k, k < n,
 * 1 <= m <= 2^24 (word (m - 1) << 8): rho_dev[k] = sqrt(-2 ln(m 2^-24)),
 * (cos_dev[k], sin_dev[k]) = (cos, sin)(pi m 2^-23), all fp64 (any may be
 * NULL), as the kernels evaluate them.  At m = 2^24 the radius comes out as
 * about 2^-200 instead of 0, which still gives a zero normal in fp32. */
CPES_API int cpes_debug_bm_grid(uint32_t m0, int64_t n, double* rho_dev, double* cos_dev,
                       double* sin_dev, void* stream);

/* The partition permutation of cpes_partition on i = i0 + k, k < n:
 * perm_dev[k] = E(i) (may be NULL), bucket_dev[k] = floor(E(i) K / d) (may be NULL). */
CPES_API int cpes_debug_prp(uint64_t seed, int64_t d, int32_t K, int64_t i0, int64_t n,
                   int64_t* perm_dev, int32_t* bucket_dev, void* stream);

/* RNG-only throughput probe: generates n normals (rounded up to a multiple
 * of 128) -- positions 0 .. n/16 - 1 of each of the 16 streams seed ..
 * seed + 15, the 16 streams of a position together as the update generates
 * its members' noise -- and folds them into sink_dev[0] (one uint32,
 * overwritten) without other memory traffic: the generator's throughput
 * when nothing else runs. */
CPES_API int cpes_rng_probe(uint64_t seed, int64_t n, uint32_t* sink_dev, void* stream);

/* Measurement references for the map and copy kernels: the same memory
 * traffic with nothing else, timed beside them.
 * cpes_probe_map_copy: the plainest gather (direction 0: buf[j] = w[p(j)])
 *   or scatter (direction 1: w[p(j)] = buf[j]) through the element map of
 *   `s` (index or index32; no chunk lists), one position per thread.  buf_dev:
 *   s->length elements of `dtype`, device memory.  Entries outside
 *   [0, numel) are skipped.
 * cpes_probe_copy: dst[i] = src[i] over `bytes` bytes (a multiple of 16; both
 *   pointers 16-byte aligned device memory), one 16-byte vector per thread;
 *   nontemporal != 0 takes non-temporal loads and stores (streaming past the
 *   caches, as the library's large copies do).
 * Errors: null pointers, a subspace without an element map, direction not 0
 *   or 1, bytes negative or not a multiple of 16, misaligned pointers ->
 *   CPES_ERR_INVALID_ARGUMENT. */
CPES_API int cpes_probe_map_copy(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, void* buf_dev,
                                 int direction, void* stream);
CPES_API int cpes_probe_copy(const void* src_dev, void* dst_dev, int64_t bytes, int nontemporal, void* stream);

/* Message of the last error on the calling thread ("" if none). */
CPES_API const char* cpes_last_error(void);

/*
 * cpes_fill_normal -- w[j] = cast(stddev * z_j) for j < n, where z_j is the
 * normal of position j in stream (seed, domain): the Philox4x32-10 words of
 * counter (lo32 q, hi32 q, domain, 0), q = j / 4, through the Box-Muller
 * transform of the perturbation noise (domain 0 is the noise itself; domain
 * 1 is meant for synthetic weight initialisation).  One fp32 multiply, then
 * round-to-nearest-even for bf16.  A utility for seeded inputs; not on the
 * training path.
 *   w_dev: n elements of `dtype` (any alignment), owned by the caller.
 * Errors: dtype unknown, n < 0, stddev negative or not finite, w NULL with
 *   n > 0 -> CPES_ERR_INVALID_ARGUMENT.  n = 0 does nothing.
 */
CPES_API int cpes_fill_normal(void* w_dev, int64_t n, int dtype, uint64_t seed, uint32_t domain, float stddev,
                     void* stream);

/* CPES_ABI_VERSION of the built library. */
CPES_API int cpes_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CPES_H */
