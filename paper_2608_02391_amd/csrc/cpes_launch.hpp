// cpes_launch.hpp -- argument blocks and launchers shared by the host runtime
// (cpes_api.hip) and the kernels (cpes_kernels.hip).  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cpes {

constexpr int kBlock = 256;             // threads per workgroup for streaming kernels
constexpr int64_t kMaxGrid = 1 << 20;   // workgroups per launch; larger jobs loop
// Workgroups per launch of the noise kernels on contiguous and chunked
// subspaces, which stage the 12 KiB Box-Muller tables (sizeof(BmTables)) in
// LDS per workgroup: a few per CU, each looping over many units.
constexpr int64_t kRngMaxGrid = 8192;

// Subspace addressing modes (see cpes_subspace).  kAddrGather32 reads a
// uint32 map through the same `index` pointer, reinterpreted.
enum AddrMode { kAddrContig = 0, kAddrGather = 1, kAddrChunk = 2, kAddrGather32 = 3 };

// One subspace operation: positions j in [0, length) at parameter offset + j,
// index[offset + j], or index[offset + j / 2^s] * 2^s + j mod 2^s (chunks).
struct StreamArgs {
    void* w;
    const int64_t* index;   // null: contiguous; a uint32 map for kAddrGather32
    void* aux;              // snapshot / backup (dtype of w) or fp32 master, may be null
    int64_t offset;
    int64_t length;
    int64_t numel;
    uint32_t k0, k1;        // Philox key = member seed
    float scale;            // +-sigma applied to the noise
    int32_t chunk_shift;    // s for chunked subspaces
    int64_t noise0;         // noise index of position 0 (a shard of a larger subspace)
    int32_t dense;          // an ascending element map: bf16 kernels may use whole-line windows
};

enum AuxKind { kAuxNone = 0, kAuxSnapshot = 1, kAuxMaster = 2, kAuxBackup = 3 };

// Update: up to kMaxMembers members folded into up to kMaxMembers distinct
// noise streams; all of it travels in the kernel argument block.
constexpr int kMaxMembers = 256;

struct UpdateArgs {
    void* w;
    const int64_t* index;
    float* master;
    const float* rnorm;
    int64_t offset;
    int64_t length;
    int64_t numel;
    float step;
    int32_t n_members;
    int32_t n_streams;
    int32_t chunk_shift;
    int64_t noise0;         // noise index of position 0
    uint32_t seed_lo[kMaxMembers];
    uint32_t seed_hi[kMaxMembers];
    uint8_t member_stream[kMaxMembers];
    int8_t member_sign[kMaxMembers];
};

// Whole-step update: every subspace of a partition with its own members, one
// launch.  Waves take tiles of 64 units from a single subspace, so the
// subspace (and its noise streams) is uniform across a wave.
constexpr int kMaxStepSubspaces = 32;

struct StepArgs {
    void* w;
    const int64_t* index;                          // null: contiguous (a uint32 map travels in this pointer)
    const float* rnorm;
    int64_t numel;
    int32_t K;
    int32_t n_members;
    int32_t n_streams;
    int32_t chunk_shift;
    uint32_t vec_mask;                             // bit k: subspace k takes 16-byte vectors
    int64_t offset[kMaxStepSubspaces + 1];         // subspace k starts at position / map entry offset[k]
    int64_t length[kMaxStepSubspaces];             // and has length[k] positions
    int64_t tile_begin[kMaxStepSubspaces + 1];     // first wave tile of subspace k
    int32_t stream_begin[kMaxStepSubspaces + 1];   // streams of subspace k
    float step[kMaxStepSubspaces];
    uint32_t seed_lo[kMaxMembers];
    uint32_t seed_hi[kMaxMembers];
    uint8_t member_stream[kMaxMembers];
    int8_t member_sign[kMaxMembers];
};

struct NormalizeArgs {
    const float* r;
    const int32_t* group;
    float* out;
    int32_t* status;
    int32_t n;
    int32_t n_groups;
    int32_t mode;
};

struct PartitionArgs {
    uint64_t seed;
    int64_t d;
    int32_t K;
    int32_t half_bits;      // h: the Feistel works on 2h bits
    uint8_t* bucket;        // workspace: bucket of every element
    uint32_t* counts;       // workspace: counts[k * n_tiles + tile]
    int64_t* pos;           // workspace: exclusive positions, same layout
    int64_t* block_sums;    // workspace: scan block partial sums
    int64_t n_tiles;
    int64_t* index;         // output map (int64), or
    uint32_t* index32;      // output map (uint32, d <= 2^32)
    int32_t* status;
};

// Tile of the permutation partition: one wave handles kTileItems x 64
// consecutive elements.
constexpr int kTileItems = 32;
constexpr int64_t kTile = 64 * kTileItems;
constexpr int kScanChunk = 4096;        // scan entries per workgroup

hipError_t launch_perturb(int dtype, int aux, int addr, bool vec, const StreamArgs& a, hipStream_t s);
hipError_t launch_restore_copy(int dtype, int addr, bool vec, const StreamArgs& a, hipStream_t s);
hipError_t launch_restore_master(int addr, bool vec, const StreamArgs& a, hipStream_t s);
hipError_t launch_backup_copy(int dtype, int addr, bool vec, const StreamArgs& a, hipStream_t s);
hipError_t launch_fill_normal(int dtype, void* w, int64_t n, uint64_t seed, uint32_t domain, float stddev, bool vec,
                              hipStream_t s);
hipError_t launch_stage_master(int dtype, int addr, bool vec, const StreamArgs& a, hipStream_t s);
hipError_t launch_update(int dtype, bool master, int addr, bool vec, const UpdateArgs& a, hipStream_t s);
hipError_t launch_update_step(int dtype, int addr, const StepArgs& a, hipStream_t s);
hipError_t launch_normalize(const NormalizeArgs& a, hipStream_t s);
hipError_t launch_partition(const PartitionArgs& a, hipStream_t s);
hipError_t launch_debug_philox(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks,
                               uint32_t* out, hipStream_t s);
hipError_t launch_debug_normals(uint64_t seed, int64_t j0, int64_t n, float* out, hipStream_t s);
hipError_t launch_debug_bm_grid(uint32_t m0, int64_t n, double* rho, double* c, double* sn, hipStream_t s);
hipError_t launch_debug_prp(uint64_t seed, int64_t d, int32_t K, int32_t half_bits, int64_t i0, int64_t n,
                            int64_t* perm, int32_t* bucket, hipStream_t s);
hipError_t launch_rng_probe(uint64_t seed, int64_t n, uint32_t* sink, hipStream_t s);
hipError_t launch_probe_map_copy(int dtype, int addr, int direction, const StreamArgs& a, hipStream_t s);
hipError_t launch_probe_copy(const void* src, void* dst, int64_t bytes, bool nontemporal, hipStream_t s);

}  // namespace cpes
