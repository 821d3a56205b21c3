// cpes_api.hip -- host runtime behind include/cpes.h: argument validation,
// dispatch to the gfx950 kernels, error reporting.  Every check runs before
// anything is enqueued, so a failing call has no effect; no HIP call is made
// before validation passes (the library loads and validates without a GPU).
#include "cpes.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "cpes_launch.hpp"

namespace {

thread_local std::string g_error;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

int hip_status(hipError_t e, const char* what)
{
    if (e != hipSuccess) return fail(CPES_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return CPES_OK;
}

bool aligned16(const void* p)
{
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

size_t elem_size(int dtype)
{
    return dtype == CPES_BF16 ? 2 : 4;
}

// Common checks of a subspace on a weight buffer.
int check_subspace(const void* w, int64_t numel, int dtype, const cpes_subspace* s, const char* fn)
{
    if (!w) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: weight pointer is null", fn);
    if (dtype != CPES_BF16 && dtype != CPES_F32) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown dtype %d", fn, dtype);
    if (!s) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: subspace is null", fn);
    if (numel < 0) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: numel %lld < 0", fn, (long long)numel);
    if (s->length < 0 || s->offset < 0)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: negative offset %lld or length %lld", fn, (long long)s->offset,
                    (long long)s->length);
    if (s->length > (INT64_MAX / 8) - s->offset)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: offset + length overflows", fn);
    if (s->noise_offset < 0 || (s->noise_offset & 7) != 0 || s->noise_offset > (INT64_MAX / 8) - s->length)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: noise_offset %lld is negative, not a multiple of 8 or too large",
                    fn, (long long)s->noise_offset);
    if (s->index && s->index32)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: a subspace takes an int64 or a uint32 map, not both", fn);
    if (s->index32 && s->chunk != 0)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: chunk lists are int64 maps", fn);
    if (s->flags & ~(int64_t)CPES_SUB_ASCENDING)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown subspace flags 0x%llx", fn, (unsigned long long)s->flags);
    if (!s->index && !s->index32 && s->offset + s->length > numel)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: range [%lld, %lld) exceeds numel %lld", fn, (long long)s->offset,
                    (long long)(s->offset + s->length), (long long)numel);
    if (s->chunk != 0) {
        if (!s->index) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: a chunked subspace needs its chunk map", fn);
        if (s->chunk < 8 || s->chunk > ((int64_t)1 << 30) || (s->chunk & (s->chunk - 1)) != 0)
            return fail(CPES_ERR_INVALID_ARGUMENT, "%s: chunk %lld is not a power of two in [8, 2^30]", fn,
                        (long long)s->chunk);
    }
    return CPES_OK;
}

int addr_mode(const cpes_subspace* s)
{
    if (s->index32) return cpes::kAddrGather32;
    if (!s->index) return cpes::kAddrContig;
    return s->chunk ? cpes::kAddrChunk : cpes::kAddrGather;
}

int log2_exact(int64_t x)
{
    int b = 0;
    while (((int64_t)1 << b) < x) ++b;
    return b;
}

int check_sign(int32_t sign, const char* fn)
{
    if (sign != 1 && sign != -1) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: sign %d is not +1 or -1", fn, sign);
    return CPES_OK;
}

int check_sigma(float sigma, const char* fn)
{
    if (!std::isfinite(sigma) || sigma < 0.0f)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: sigma %g is negative or not finite", fn, (double)sigma);
    return CPES_OK;
}

// Whether the 16-byte vector path applies: every unit's vectors are aligned.
// Element maps are read one entry per lane, and the weights they address one
// element at a time, so only the side buffer's alignment matters for them.
bool vector_ok(const void* w, int dtype, const cpes_subspace* s, const void* aux, bool aux_is_master)
{
    if (s->index && s->chunk) {
        if (!aligned16(w)) return false;                    // chunk starts are multiples of 8 elements
    } else if (s->index || s->index32) {
        // nothing: the map kernels take any map offset
    } else {
        const char* base = static_cast<const char*>(w) + (size_t)s->offset * elem_size(dtype);
        if (!aligned16(base)) return false;
    }
    if (aux && !aligned16(aux)) return false;
    (void)aux_is_master;
    return true;
}

cpes::StreamArgs stream_args(void* w, int64_t numel, const cpes_subspace* s, const void* aux, uint64_t seed,
                             float scale)
{
    cpes::StreamArgs a;
    a.w = w;
    a.index = s->index32 ? reinterpret_cast<const int64_t*>(s->index32) : s->index;
    a.aux = const_cast<void*>(aux);
    a.offset = s->offset;
    a.length = s->length;
    a.numel = numel;
    a.k0 = (uint32_t)seed;
    a.k1 = (uint32_t)(seed >> 32);
    a.scale = scale;
    a.chunk_shift = s->chunk ? log2_exact(s->chunk) : 0;
    a.noise0 = s->noise_offset;
    a.dense = (s->flags & CPES_SUB_ASCENDING) && (s->index32 || (s->index && !s->chunk)) ? 1 : 0;
    return a;
}

// Host replay of the partition permutation (the same definition the device
// kernels implement), used to find the subspace of one chunk.
void host_philox(uint32_t c[4], uint32_t k0, uint32_t k1)
{
    for (int r = 0; r < 10; ++r) {
        const uint64_t pa = (uint64_t)0xD2511F53u * c[0];
        const uint64_t pb = (uint64_t)0xCD9E8D57u * c[2];
        const uint32_t n0 = (uint32_t)(pb >> 32) ^ c[1] ^ k0;
        const uint32_t n2 = (uint32_t)(pa >> 32) ^ c[3] ^ k1;
        c[1] = (uint32_t)pb;
        c[3] = (uint32_t)pa;
        c[0] = n0;
        c[2] = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
}

uint64_t host_feistel(uint64_t seed, int h, uint64_t x)
{
    const uint64_t mask = (1ull << h) - 1ull;
    uint64_t L = x >> h, R = x & mask;
    for (uint32_t r = 0; r < 8; ++r) {
        uint32_t c[4] = {(uint32_t)R, r, 3u, 0u};
        host_philox(c, (uint32_t)seed, (uint32_t)(seed >> 32));
        const uint64_t nr = L ^ ((uint64_t)c[0] & mask);
        L = R;
        R = nr;
    }
    return (L << h) | R;
}

int feistel_half_bits(int64_t d)
{
    int b = 0;
    while (b < 63 && ((int64_t)1 << b) < d) ++b;
    if (b < 2) b = 2;
    if (b & 1) ++b;
    return b / 2;
}

struct PartitionLayout {
    int64_t n_tiles, n_counts, scan_blocks;
    size_t off_counts, off_pos, off_block_sums, total;
};

constexpr size_t round_up(size_t x, size_t a)
{
    return (x + a - 1) / a * a;
}

constexpr PartitionLayout partition_layout(int64_t d, int32_t K)
{
    PartitionLayout L{};
    L.n_tiles = (d + cpes::kTile - 1) / cpes::kTile;
    L.n_counts = (int64_t)K * L.n_tiles;
    L.scan_blocks = (L.n_counts + cpes::kScanChunk - 1) / cpes::kScanChunk;
    L.off_counts = round_up((size_t)d, 256);
    L.off_pos = round_up(L.off_counts + (size_t)L.n_counts * 4, 256);
    L.off_block_sums = round_up(L.off_pos + (size_t)L.n_counts * 8, 256);
    L.total = round_up(L.off_block_sums + (size_t)L.scan_blocks * 8, 256);
    return L;
}

// ------------------------------------------ allocation-free chunk partition --
// cpes_partition_chunks_static takes its workspace from this file-scope device
// array instead of a caller's buffer, sized for the largest partition it
// accepts.  Each GPU holds its own copy until the process ends; host code
// never passes the array's name to a kernel (on the host it is only a
// stand-in symbol) but the device address that hipGetSymbolAddress returns,
// looked up once per device on the first call there.
constexpr size_t kStaticScratchBytes = partition_layout(CPES_STATIC_MAX_CHUNKS, CPES_MAX_PERMUTATION_K).total;
static_assert(kStaticScratchBytes == 2621696, "the size include/cpes.h states");
static __device__ __attribute__((aligned(256))) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once looked up

int static_scratch(void** ws, const char* fn)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, fn);
    if (dev < 0 || dev >= kMaxDevices)
        return fail(CPES_ERR_UNSUPPORTED, "%s: device %d beyond the %d the library tracks", fn, dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(e, fn);
        if (!p || !aligned16(p)) return fail(CPES_ERR_HIP, "%s: no usable device address for the static workspace", fn);
        g_scratch_ptr[dev] = p;
    }
    *ws = g_scratch_ptr[dev];
    return CPES_OK;
}

int check_chunk_partition(int64_t d, int64_t chunk, int32_t K, const int64_t* list_offsets_host,
                          const int64_t* lengths_host, const char* fn);
int chunk_partition(int64_t d, int64_t chunk, int32_t K, uint64_t seed, int64_t* list_offsets_host,
                    int64_t* lengths_host, int64_t* chunks_dev, void* workspace_dev, size_t workspace_bytes,
                    int32_t* status_dev, void* stream, const char* fn);

// The keyed-permutation partition into an int64 or a uint32 map.
int permutation_partition(int64_t d, int32_t K, uint64_t seed, int64_t* offsets_host, int64_t* index64,
                          uint32_t* index32, void* workspace_dev, size_t workspace_bytes, int32_t* status_dev,
                          void* stream, const char* fn)
{
    if (K > CPES_MAX_PERMUTATION_K)
        return fail(CPES_ERR_UNSUPPORTED, "%s: K %d above CPES_MAX_PERMUTATION_K", fn, K);
    if (d >= ((int64_t)1 << 55)) return fail(CPES_ERR_UNSUPPORTED, "%s: permutation needs d < 2^55", fn);
    const PartitionLayout L = partition_layout(d, K);
    if (!workspace_dev || workspace_bytes < L.total)
        return fail(CPES_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, L.total,
                    workspace_dev ? workspace_bytes : (size_t)0);
    if (!aligned16(workspace_dev)) return fail(CPES_ERR_WORKSPACE, "%s: workspace must be 16-byte aligned", fn);
    for (int32_t k = 0; k <= K; ++k)
        offsets_host[k] = (int64_t)(((unsigned __int128)(uint64_t)d * (uint64_t)k + (uint64_t)K - 1u) / (uint64_t)K);
    char* ws = static_cast<char*>(workspace_dev);
    cpes::PartitionArgs a;
    a.seed = seed;
    a.d = d;
    a.K = K;
    a.half_bits = feistel_half_bits(d);
    a.bucket = reinterpret_cast<uint8_t*>(ws);
    a.counts = reinterpret_cast<uint32_t*>(ws + L.off_counts);
    a.pos = reinterpret_cast<int64_t*>(ws + L.off_pos);
    a.block_sums = reinterpret_cast<int64_t*>(ws + L.off_block_sums);
    a.n_tiles = L.n_tiles;
    a.index = index64;
    a.index32 = index32;
    a.status = status_dev;
    return hip_status(cpes::launch_partition(a, (hipStream_t)stream), fn);
}

// A host backup must be pinned memory the device can address (hipHostMalloc,
// torch pin_memory); a kernel touching pageable memory would fault.  Returns
// the device-side address of the buffer in *dev.
int check_pinned_host(const void* p, void** dev, const char* fn)
{
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess || attr.type != hipMemoryTypeHost) {
        (void)hipGetLastError();
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: the backup is not pinned host memory", fn);
    }
    *dev = attr.devicePointer ? attr.devicePointer : const_cast<void*>(p);
    return CPES_OK;
}

int host_backup_copy(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, void* host, bool to_host,
                     void* stream, const char* fn)
{
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if (!host) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: backup pointer is null", fn);
    if (s->length == 0) return CPES_OK;
    void* host_dev = nullptr;
    if ((rc = check_pinned_host(host, &host_dev, fn))) return rc;
    hipStream_t st = (hipStream_t)stream;
    if (!s->index && !s->index32) {   // contiguous: one DMA transfer over the host link
        const size_t bytes = (size_t)s->length * elem_size(dtype);
        char* dev = static_cast<char*>(w_dev) + (size_t)s->offset * elem_size(dtype);
        const hipError_t e = to_host ? hipMemcpyAsync(host, dev, bytes, hipMemcpyDeviceToHost, st)
                                     : hipMemcpyAsync(dev, host, bytes, hipMemcpyHostToDevice, st);
        return hip_status(e, fn);
    }
    // index-map or chunked: the copy kernels address the pinned buffer directly
    const cpes::StreamArgs a = stream_args(w_dev, numel, s, host_dev, 0, 0.0f);
    const bool vec = vector_ok(w_dev, dtype, s, host_dev, false);
    if (to_host) return hip_status(cpes::launch_backup_copy(dtype, addr_mode(s), vec, a, st), fn);
    return hip_status(cpes::launch_restore_copy(dtype, addr_mode(s), vec, a, st), fn);
}

}  // namespace

extern "C" {

const char* cpes_last_error(void)
{
    return g_error.c_str();
}

int cpes_abi_version(void)
{
    return CPES_ABI_VERSION;
}

size_t cpes_partition_workspace_bytes(int mode, int64_t d, int32_t K)
{
    if (mode == CPES_PART_CONTIGUOUS) return 0;
    if (mode != CPES_PART_PERMUTATION || d < 1 || K < 1 || K > CPES_MAX_PERMUTATION_K || (int64_t)K > d ||
        d >= ((int64_t)1 << 55))
        return 0;
    return partition_layout(d, K).total;
}

int cpes_partition(int mode, int64_t d, int32_t K, uint64_t seed, const int64_t* bounds_host, int64_t* offsets_host,
                   int64_t* index_dev, void* workspace_dev, size_t workspace_bytes, int32_t* status_dev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_partition";
    if (mode != CPES_PART_CONTIGUOUS && mode != CPES_PART_PERMUTATION)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown mode %d", fn, mode);
    if (d < 1 || d >= ((int64_t)1 << 62)) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: d %lld out of range", fn, (long long)d);
    if (K < 1 || (int64_t)K > d) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: K %d not in [1, d]", fn, K);
    if (!offsets_host) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: offsets_host is null", fn);
    if (mode == CPES_PART_CONTIGUOUS) {
        if (bounds_host) {
            if (bounds_host[0] != 0 || bounds_host[K] != d)
                return fail(CPES_ERR_INVALID_ARGUMENT, "%s: bounds must run from 0 to d", fn);
            for (int32_t k = 0; k < K; ++k)
                if (bounds_host[k + 1] < bounds_host[k])
                    return fail(CPES_ERR_INVALID_ARGUMENT, "%s: bounds decrease at %d", fn, k);
            for (int32_t k = 0; k <= K; ++k) offsets_host[k] = bounds_host[k];
        } else {
            for (int32_t k = 0; k <= K; ++k)
                offsets_host[k] = (int64_t)(((unsigned __int128)(uint64_t)d * (uint64_t)k) / (uint64_t)K);
        }
        return CPES_OK;
    }
    if (!index_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: index_dev is null", fn);
    return permutation_partition(d, K, seed, offsets_host, index_dev, nullptr, workspace_dev, workspace_bytes,
                                 status_dev, stream, fn);
}

int cpes_partition32(int64_t d, int32_t K, uint64_t seed, int64_t* offsets_host, uint32_t* index_dev,
                     void* workspace_dev, size_t workspace_bytes, int32_t* status_dev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_partition32";
    if (d < 1 || d > ((int64_t)1 << 32))
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: d %lld not in [1, 2^32]", fn, (long long)d);
    if (K < 1 || (int64_t)K > d) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: K %d not in [1, d]", fn, K);
    if (!offsets_host) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: offsets_host is null", fn);
    if (!index_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: index_dev is null", fn);
    return permutation_partition(d, K, seed, offsets_host, nullptr, index_dev, workspace_dev, workspace_bytes,
                                 status_dev, stream, fn);
}

size_t cpes_partition_chunks_workspace_bytes(int64_t d, int64_t chunk, int32_t K)
{
    if (d < 1 || chunk < 8 || chunk > ((int64_t)1 << 30) || (chunk & (chunk - 1)) != 0) return 0;
    const int64_t n_chunks = (d + chunk - 1) / chunk;
    return cpes_partition_workspace_bytes(CPES_PART_PERMUTATION, n_chunks, K);
}

int cpes_partition_chunks(int64_t d, int64_t chunk, int32_t K, uint64_t seed, int64_t* list_offsets_host,
                          int64_t* lengths_host, int64_t* chunks_dev, void* workspace_dev, size_t workspace_bytes,
                          int32_t* status_dev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_partition_chunks";
    int rc = check_chunk_partition(d, chunk, K, list_offsets_host, lengths_host, fn);
    if (rc) return rc;
    return chunk_partition(d, chunk, K, seed, list_offsets_host, lengths_host, chunks_dev, workspace_dev,
                           workspace_bytes, status_dev, stream, fn);
}

int cpes_partition_chunks_static(int64_t d, int64_t chunk, int32_t K, uint64_t seed, int64_t* list_offsets_host,
                                 int64_t* lengths_host, int64_t* chunks_dev, int32_t* status_dev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_partition_chunks_static";
    int rc = check_chunk_partition(d, chunk, K, list_offsets_host, lengths_host, fn);
    if (rc) return rc;
    const int64_t n_chunks = (d + chunk - 1) / chunk;
    if (n_chunks > CPES_STATIC_MAX_CHUNKS || K > CPES_MAX_PERMUTATION_K)
        return fail(CPES_ERR_UNSUPPORTED, "%s: %lld chunks and K %d exceed the static workspace (at most %d chunks, "
                    "K <= %d); use cpes_partition_chunks with a workspace", fn, (long long)n_chunks, K,
                    CPES_STATIC_MAX_CHUNKS, CPES_MAX_PERMUTATION_K);
    void* ws = nullptr;
    if ((rc = static_scratch(&ws, fn))) return rc;
    return chunk_partition(d, chunk, K, seed, list_offsets_host, lengths_host, chunks_dev, ws, kStaticScratchBytes,
                           status_dev, stream, fn);
}

}  // extern "C"

namespace {

int check_chunk_partition(int64_t d, int64_t chunk, int32_t K, const int64_t* list_offsets_host,
                          const int64_t* lengths_host, const char* fn)
{
    if (d < 1 || d >= ((int64_t)1 << 62)) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: d %lld out of range", fn, (long long)d);
    if (chunk < 8 || chunk > ((int64_t)1 << 30) || (chunk & (chunk - 1)) != 0)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: chunk %lld is not a power of two in [8, 2^30]", fn, (long long)chunk);
    if (!list_offsets_host || !lengths_host) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: null host outputs", fn);
    const int64_t n_chunks = (d + chunk - 1) / chunk;
    if (K < 1 || (int64_t)K > n_chunks)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: K %d not in [1, %lld chunks]", fn, K, (long long)n_chunks);
    return CPES_OK;
}

// The chunk partition after argument checks, on the given workspace.
int chunk_partition(int64_t d, int64_t chunk, int32_t K, uint64_t seed, int64_t* list_offsets_host,
                    int64_t* lengths_host, int64_t* chunks_dev, void* workspace_dev, size_t workspace_bytes,
                    int32_t* status_dev, void* stream, const char* fn)
{
    const int64_t n_chunks = (d + chunk - 1) / chunk;
    // the chunk permutation is the permutation partition of the chunk ids
    int rc = cpes_partition(CPES_PART_PERMUTATION, n_chunks, K, seed, nullptr, list_offsets_host, chunks_dev,
                            workspace_dev, workspace_bytes, status_dev, stream);
    if (rc) {
        const std::string msg = g_error;
        return fail(rc, "%s: %s", fn, msg.c_str());
    }
    for (int32_t k = 0; k < K; ++k) lengths_host[k] = (list_offsets_host[k + 1] - list_offsets_host[k]) * chunk;
    const int64_t short_by = n_chunks * chunk - d;
    if (short_by > 0) {   // the last chunk is short; find its subspace
        const int h = feistel_half_bits(n_chunks);
        uint64_t y = host_feistel(seed, h, (uint64_t)(n_chunks - 1));
        while (y >= (uint64_t)n_chunks) y = host_feistel(seed, h, y);
        const int32_t k = (int32_t)((y * (uint64_t)K) / (uint64_t)n_chunks);
        lengths_host[k] -= short_by;
    }
    return CPES_OK;
}

}  // namespace

extern "C" {

int cpes_perturb(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float sigma, uint64_t seed,
                 int32_t sign, void* aux_dev, int aux_mode, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_perturb";
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if ((rc = check_sign(sign, fn)) || (rc = check_sigma(sigma, fn))) return rc;
    if (aux_mode != CPES_AUX_NONE && aux_mode != CPES_AUX_SNAPSHOT && aux_mode != CPES_AUX_MASTER &&
        aux_mode != CPES_AUX_BACKUP)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown aux_mode %d", fn, aux_mode);
    if (aux_mode != CPES_AUX_NONE && !aux_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: aux buffer is null", fn);
    if (aux_mode == CPES_AUX_MASTER && dtype != CPES_BF16)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: master source needs bf16 weights", fn);
    if (s->length == 0) return CPES_OK;
    const float scale = sign > 0 ? sigma : -sigma;
    const void* aux = aux_mode == CPES_AUX_NONE ? nullptr : aux_dev;
    const bool vec = vector_ok(w_dev, dtype, s, aux, aux_mode == CPES_AUX_MASTER);
    const cpes::StreamArgs a = stream_args(w_dev, numel, s, aux, seed, scale);
    return hip_status(cpes::launch_perturb(dtype, aux_mode, addr_mode(s), vec, a, (hipStream_t)stream), fn);
}

int cpes_restore(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float sigma, uint64_t seed,
                 int32_t sign, const void* aux_dev, int aux_mode, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_restore";
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if (aux_mode != CPES_AUX_NONE && aux_mode != CPES_AUX_SNAPSHOT && aux_mode != CPES_AUX_MASTER)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown aux_mode %d", fn, aux_mode);
    if (aux_mode == CPES_AUX_NONE) {
        if ((rc = check_sign(sign, fn)) || (rc = check_sigma(sigma, fn))) return rc;
    } else if (!aux_dev) {
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: aux buffer is null", fn);
    }
    if (aux_mode == CPES_AUX_MASTER && dtype != CPES_BF16)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: master source needs bf16 weights", fn);
    if (s->length == 0) return CPES_OK;
    const int addr = addr_mode(s);
    hipStream_t st = (hipStream_t)stream;
    if (aux_mode == CPES_AUX_NONE) {
        const float scale = sign > 0 ? -sigma : sigma;
        const cpes::StreamArgs a = stream_args(w_dev, numel, s, nullptr, seed, scale);
        return hip_status(cpes::launch_perturb(dtype, cpes::kAuxNone, addr, vector_ok(w_dev, dtype, s, nullptr, false), a, st), fn);
    }
    const cpes::StreamArgs a = stream_args(w_dev, numel, s, aux_dev, seed, 0.0f);
    const bool vec = vector_ok(w_dev, dtype, s, aux_dev, aux_mode == CPES_AUX_MASTER);
    if (aux_mode == CPES_AUX_SNAPSHOT) return hip_status(cpes::launch_restore_copy(dtype, addr, vec, a, st), fn);
    return hip_status(cpes::launch_restore_master(addr, vec, a, st), fn);
}

int cpes_backup_to_host(const void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, void* backup_host,
                        void* stream)
{
    g_error.clear();
    return host_backup_copy(const_cast<void*>(w_dev), numel, dtype, s, backup_host, true, stream,
                            "cpes_backup_to_host");
}

int cpes_restore_from_host(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, const void* backup_host,
                           void* stream)
{
    g_error.clear();
    return host_backup_copy(w_dev, numel, dtype, s, const_cast<void*>(backup_host), false, stream,
                            "cpes_restore_from_host");
}

int cpes_backup(const void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, void* backup_dev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_backup";
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if (!backup_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: backup pointer is null", fn);
    if (s->length == 0) return CPES_OK;
    const cpes::StreamArgs a = stream_args(const_cast<void*>(w_dev), numel, s, backup_dev, 0, 0.0f);
    const bool vec = vector_ok(w_dev, dtype, s, backup_dev, false);
    return hip_status(cpes::launch_backup_copy(dtype, addr_mode(s), vec, a, (hipStream_t)stream), fn);
}

int cpes_stage_master(const void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float* master_dev,
                      void* stream)
{
    g_error.clear();
    const char* fn = "cpes_stage_master";
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if (!master_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: master_dev is null", fn);
    if (s->length == 0) return CPES_OK;
    const bool vec = vector_ok(w_dev, dtype, s, master_dev, true);
    const cpes::StreamArgs a = stream_args(const_cast<void*>(w_dev), numel, s, master_dev, 0, 0.0f);
    return hip_status(cpes::launch_stage_master(dtype, addr_mode(s), vec, a, (hipStream_t)stream), fn);
}

int cpes_normalize_rewards(const float* r_dev, int32_t n, int mode, const int32_t* group_dev, int32_t n_groups,
                           float* out_dev, int32_t* status_dev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_normalize_rewards";
    if (!r_dev || !out_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: null reward or output pointer", fn);
    if (n < 1 || n > CPES_MAX_REWARDS) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: n %d not in [1, %d]", fn, n, CPES_MAX_REWARDS);
    if (mode != CPES_NORM_Z && mode != CPES_NORM_RANK) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown mode %d", fn, mode);
    if (group_dev) {
        if (n_groups < 1 || n_groups > n)
            return fail(CPES_ERR_INVALID_ARGUMENT, "%s: n_groups %d not in [1, n]", fn, n_groups);
        if (n_groups > CPES_MAX_GROUPS)
            return fail(CPES_ERR_UNSUPPORTED, "%s: n_groups %d above CPES_MAX_GROUPS", fn, n_groups);
    }
    cpes::NormalizeArgs a;
    a.r = r_dev;
    a.group = group_dev;
    a.out = out_dev;
    a.status = status_dev;
    a.n = n;
    a.n_groups = group_dev ? n_groups : 1;
    a.mode = mode;
    return hip_status(cpes::launch_normalize(a, (hipStream_t)stream), fn);
}

int cpes_update(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, float* master_dev, int32_t n,
                const uint64_t* seeds_host, const int8_t* signs_host, const float* rnorm_dev, float alpha, float sigma,
                int scale_mode, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_update";
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if (n < 1) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: n %d < 1", fn, n);
    if (n > CPES_MAX_MEMBERS) return fail(CPES_ERR_UNSUPPORTED, "%s: n %d above CPES_MAX_MEMBERS", fn, n);
    if (!seeds_host || !signs_host || !rnorm_dev)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: null seeds, signs or rewards", fn);
    if (scale_mode != CPES_SCALE_ALPHA_OVER_N_SIGMA && scale_mode != CPES_SCALE_ALPHA_OVER_N)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown scale_mode %d", fn, scale_mode);
    if (!std::isfinite(alpha)) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: alpha is not finite", fn);
    if (scale_mode == CPES_SCALE_ALPHA_OVER_N_SIGMA && (!std::isfinite(sigma) || sigma <= 0.0f))
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: sigma %g must be finite and > 0", fn, (double)sigma);
    if (master_dev && dtype != CPES_BF16)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: a master copy needs bf16 weights", fn);
    cpes::UpdateArgs a;
    std::memset(&a, 0, sizeof a);
    int n_streams = 0;
    for (int32_t i = 0; i < n; ++i) {
        if ((rc = check_sign(signs_host[i], fn))) return rc;
        int u = 0;
        while (u < n_streams && ((uint64_t)a.seed_lo[u] | ((uint64_t)a.seed_hi[u] << 32)) != seeds_host[i]) ++u;
        if (u == n_streams) {
            a.seed_lo[u] = (uint32_t)seeds_host[i];
            a.seed_hi[u] = (uint32_t)(seeds_host[i] >> 32);
            ++n_streams;
        }
        a.member_stream[i] = (uint8_t)u;
        a.member_sign[i] = signs_host[i];
    }
    if (s->length == 0) return CPES_OK;
    const double step = scale_mode == CPES_SCALE_ALPHA_OVER_N_SIGMA ? (double)alpha / ((double)n * (double)sigma)
                                                                    : (double)alpha / (double)n;
    a.w = w_dev;
    a.index = s->index32 ? reinterpret_cast<const int64_t*>(s->index32) : s->index;
    a.master = master_dev;
    a.rnorm = rnorm_dev;
    a.offset = s->offset;
    a.length = s->length;
    a.numel = numel;
    a.step = (float)step;
    a.n_members = n;
    a.n_streams = n_streams;
    a.chunk_shift = s->chunk ? log2_exact(s->chunk) : 0;
    a.noise0 = s->noise_offset;
    const bool vec = vector_ok(w_dev, dtype, s, master_dev, true);
    return hip_status(cpes::launch_update(dtype, master_dev != nullptr, addr_mode(s), vec, a, (hipStream_t)stream), fn);
}

}  // extern "C"

namespace {

// cpes_update_step and cpes_update_step32: the map is int64 entries (or chunk
// ids), or uint32 entries when idx32.
int update_step_impl(void* w_dev, int64_t numel, int dtype, int32_t K, const int64_t* offsets_host,
                     const void* index_dev, bool idx32, int64_t chunk, const int64_t* lengths_host, int32_t n,
                     const uint64_t* seeds_host, const int8_t* signs_host, const int32_t* subspace_host,
                     const float* rnorm_dev, float alpha, const float* sigma_host, int scale_mode, void* stream,
                     const char* fn)
{
    if (!w_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: weight pointer is null", fn);
    if (dtype != CPES_BF16 && dtype != CPES_F32) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown dtype %d", fn, dtype);
    if (K < 1) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: K %d < 1", fn, K);
    if (K > CPES_MAX_STEP_SUBSPACES) return fail(CPES_ERR_UNSUPPORTED, "%s: K %d above CPES_MAX_STEP_SUBSPACES", fn, K);
    if (!offsets_host || !seeds_host || !signs_host || !subspace_host || !rnorm_dev || !sigma_host)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: null offsets, members, rewards or sigmas", fn);
    if (n < 1) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: n %d < 1", fn, n);
    if (n > CPES_MAX_MEMBERS) return fail(CPES_ERR_UNSUPPORTED, "%s: n %d above CPES_MAX_MEMBERS", fn, n);
    if (scale_mode != CPES_SCALE_ALPHA_OVER_N_SIGMA && scale_mode != CPES_SCALE_ALPHA_OVER_N)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown scale_mode %d", fn, scale_mode);
    if (!std::isfinite(alpha)) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: alpha is not finite", fn);
    if (offsets_host[0] < 0) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: offsets[0] < 0", fn);
    if (chunk != 0) {
        if (!index_dev || !lengths_host)
            return fail(CPES_ERR_INVALID_ARGUMENT, "%s: chunked subspaces need the chunk map and lengths", fn);
        if (chunk < 8 || chunk > ((int64_t)1 << 30) || (chunk & (chunk - 1)) != 0)
            return fail(CPES_ERR_INVALID_ARGUMENT, "%s: chunk %lld is not a power of two in [8, 2^30]", fn, (long long)chunk);
        for (int32_t k = 0; k < K; ++k)
            if (lengths_host[k] < 0 || lengths_host[k] > (offsets_host[k + 1] - offsets_host[k]) * chunk)
                return fail(CPES_ERR_INVALID_ARGUMENT, "%s: length of subspace %d does not fit its chunks", fn, k);
    }
    for (int32_t k = 0; k < K; ++k)
        if (offsets_host[k + 1] < offsets_host[k]) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: offsets decrease at %d", fn, k);
    if (!index_dev && offsets_host[K] > numel)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: offsets[K] %lld exceeds numel %lld", fn, (long long)offsets_host[K],
                    (long long)numel);
    int count[CPES_MAX_STEP_SUBSPACES] = {0};
    for (int32_t i = 0; i < n; ++i) {
        int rc = check_sign(signs_host[i], fn);
        if (rc) return rc;
        if (subspace_host[i] < 0 || subspace_host[i] >= K)
            return fail(CPES_ERR_INVALID_ARGUMENT, "%s: member %d names subspace %d", fn, i, subspace_host[i]);
        ++count[subspace_host[i]];
    }
    cpes::StepArgs a;
    std::memset(&a, 0, sizeof a);
    // streams: distinct (subspace, seed) pairs, grouped by subspace, in order of first appearance
    int n_streams = 0;
    for (int32_t k = 0; k < K; ++k) {
        a.stream_begin[k] = n_streams;
        for (int32_t i = 0; i < n; ++i) {
            if (subspace_host[i] != k) continue;
            int u = a.stream_begin[k];
            while (u < n_streams && ((uint64_t)a.seed_lo[u] | ((uint64_t)a.seed_hi[u] << 32)) != seeds_host[i]) ++u;
            if (u == n_streams) {
                a.seed_lo[u] = (uint32_t)seeds_host[i];
                a.seed_hi[u] = (uint32_t)(seeds_host[i] >> 32);
                ++n_streams;
            }
            a.member_stream[i] = (uint8_t)u;
            a.member_sign[i] = signs_host[i];
        }
        if (count[k] > 0) {
            const float sig = sigma_host[k];
            if (scale_mode == CPES_SCALE_ALPHA_OVER_N_SIGMA && (!std::isfinite(sig) || sig <= 0.0f))
                return fail(CPES_ERR_INVALID_ARGUMENT, "%s: sigma[%d] %g must be finite and > 0", fn, k, (double)sig);
            const double step = scale_mode == CPES_SCALE_ALPHA_OVER_N_SIGMA
                                    ? (double)alpha / ((double)count[k] * (double)sig)
                                    : (double)alpha / (double)count[k];
            a.step[k] = (float)step;
        }
    }
    a.stream_begin[K] = n_streams;
    const int N = dtype == CPES_BF16 ? 8 : 4;
    int64_t tiles = 0;
    for (int32_t k = 0; k <= K; ++k) {
        a.offset[k] = offsets_host[k];
        a.tile_begin[k] = tiles;
        if (k == K) break;
        const int64_t len = chunk ? lengths_host[k] : offsets_host[k + 1] - offsets_host[k];
        a.length[k] = len;
        const int64_t units = (len + N - 1) / N;
        if (count[k] > 0) tiles += (units + 63) / 64;   // subspaces without members are left alone
        const void* first = chunk ? w_dev
                          : index_dev ? (const void*)(static_cast<const char*>(index_dev) +
                                                      (size_t)offsets_host[k] * (idx32 ? 4 : 8))
                                      : (const void*)(static_cast<const char*>(w_dev) + (size_t)offsets_host[k] * elem_size(dtype));
        if (aligned16(first)) a.vec_mask |= 1u << k;
    }
    a.chunk_shift = chunk ? log2_exact(chunk) : 0;
    a.w = w_dev;
    a.index = static_cast<const int64_t*>(index_dev);
    a.rnorm = rnorm_dev;
    a.numel = numel;
    a.K = K;
    a.n_members = n;
    a.n_streams = n_streams;
    if (tiles == 0) return CPES_OK;
    const int addr = !index_dev ? cpes::kAddrContig
                   : idx32      ? cpes::kAddrGather32
                   : chunk      ? cpes::kAddrChunk
                                : cpes::kAddrGather;
    return hip_status(cpes::launch_update_step(dtype, addr, a, (hipStream_t)stream), fn);
}

}  // namespace

extern "C" {

int cpes_update_step(void* w_dev, int64_t numel, int dtype, int32_t K, const int64_t* offsets_host,
                     const int64_t* index_dev, int64_t chunk, const int64_t* lengths_host, int32_t n,
                     const uint64_t* seeds_host, const int8_t* signs_host,
                     const int32_t* subspace_host, const float* rnorm_dev, float alpha, const float* sigma_host,
                     int scale_mode, void* stream)
{
    g_error.clear();
    return update_step_impl(w_dev, numel, dtype, K, offsets_host, index_dev, false, chunk, lengths_host, n,
                            seeds_host, signs_host, subspace_host, rnorm_dev, alpha, sigma_host, scale_mode, stream,
                            "cpes_update_step");
}

int cpes_update_step32(void* w_dev, int64_t numel, int dtype, int32_t K, const int64_t* offsets_host,
                       const uint32_t* index32_dev, int32_t n, const uint64_t* seeds_host, const int8_t* signs_host,
                       const int32_t* subspace_host, const float* rnorm_dev, float alpha, const float* sigma_host,
                       int scale_mode, void* stream)
{
    g_error.clear();
    if (!index32_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "cpes_update_step32: index32 map is null");
    return update_step_impl(w_dev, numel, dtype, K, offsets_host, index32_dev, true, 0, nullptr, n, seeds_host,
                            signs_host, subspace_host, rnorm_dev, alpha, sigma_host, scale_mode, stream,
                            "cpes_update_step32");
}

int cpes_fill_normal(void* w_dev, int64_t n, int dtype, uint64_t seed, uint32_t domain, float stddev, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_fill_normal";
    if (dtype != CPES_BF16 && dtype != CPES_F32) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: unknown dtype %d", fn, dtype);
    if (n < 0) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: n %lld is negative", fn, (long long)n);
    int rc = check_sigma(stddev, fn);
    if (rc) return rc;
    if (n == 0) return CPES_OK;
    if (!w_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: w is null", fn);
    return hip_status(cpes::launch_fill_normal(dtype, w_dev, n, seed, domain, stddev, aligned16(w_dev),
                                               (hipStream_t)stream), fn);
}

int cpes_debug_philox(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks, uint32_t* out_dev, void* stream)
{
    g_error.clear();
    if (!out_dev || nblocks < 0) return fail(CPES_ERR_INVALID_ARGUMENT, "cpes_debug_philox: bad output or count");
    if (nblocks == 0) return CPES_OK;
    return hip_status(cpes::launch_debug_philox(seed, domain, q0, nblocks, out_dev, (hipStream_t)stream), "cpes_debug_philox");
}

int cpes_debug_normals(uint64_t seed, int64_t j0, int64_t n, float* out_dev, void* stream)
{
    g_error.clear();
    if (!out_dev || n < 0 || j0 < 0) return fail(CPES_ERR_INVALID_ARGUMENT, "cpes_debug_normals: bad output, j0 or count");
    if (n == 0) return CPES_OK;
    return hip_status(cpes::launch_debug_normals(seed, j0, n, out_dev, (hipStream_t)stream), "cpes_debug_normals");
}

int cpes_debug_bm_grid(uint32_t m0, int64_t n, double* rho_dev, double* cos_dev, double* sin_dev, void* stream)
{
    g_error.clear();
    if (n < 0 || m0 < 1 || (int64_t)m0 + n - 1 > ((int64_t)1 << 24))
        return fail(CPES_ERR_INVALID_ARGUMENT, "cpes_debug_bm_grid: grid outside [1, 2^24]");
    if (n == 0) return CPES_OK;
    return hip_status(cpes::launch_debug_bm_grid(m0, n, rho_dev, cos_dev, sin_dev, (hipStream_t)stream), "cpes_debug_bm_grid");
}

int cpes_debug_prp(uint64_t seed, int64_t d, int32_t K, int64_t i0, int64_t n, int64_t* perm_dev, int32_t* bucket_dev,
                   void* stream)
{
    g_error.clear();
    if (d < 1 || d >= ((int64_t)1 << 55) || K < 1 || K > CPES_MAX_PERMUTATION_K || (int64_t)K > d || i0 < 0 || n < 0 ||
        i0 + n > d)
        return fail(CPES_ERR_INVALID_ARGUMENT, "cpes_debug_prp: bad d, K or range");
    if (n == 0) return CPES_OK;
    return hip_status(cpes::launch_debug_prp(seed, d, K, feistel_half_bits(d), i0, n, perm_dev, bucket_dev,
                                             (hipStream_t)stream),
                      "cpes_debug_prp");
}

int cpes_probe_map_copy(void* w_dev, int64_t numel, int dtype, const cpes_subspace* s, void* buf_dev, int direction,
                        void* stream)
{
    g_error.clear();
    const char* fn = "cpes_probe_map_copy";
    int rc = check_subspace(w_dev, numel, dtype, s, fn);
    if (rc) return rc;
    if ((!s->index && !s->index32) || s->chunk != 0)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: needs an element map (index or index32)", fn);
    if (!buf_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: buffer is null", fn);
    if (direction != 0 && direction != 1)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: direction %d is not 0 (gather) or 1 (scatter)", fn, direction);
    if (s->length == 0) return CPES_OK;
    const cpes::StreamArgs a = stream_args(w_dev, numel, s, buf_dev, 0, 0.0f);
    return hip_status(cpes::launch_probe_map_copy(dtype, addr_mode(s), direction, a, (hipStream_t)stream), fn);
}

int cpes_probe_copy(const void* src_dev, void* dst_dev, int64_t bytes, int nontemporal, void* stream)
{
    g_error.clear();
    const char* fn = "cpes_probe_copy";
    if (!src_dev || !dst_dev) return fail(CPES_ERR_INVALID_ARGUMENT, "%s: null pointer", fn);
    if (bytes < 0 || (bytes & 15) != 0)
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: bytes %lld is negative or not a multiple of 16", fn, (long long)bytes);
    if (!aligned16(src_dev) || !aligned16(dst_dev))
        return fail(CPES_ERR_INVALID_ARGUMENT, "%s: pointers must be 16-byte aligned", fn);
    if (bytes == 0) return CPES_OK;
    return hip_status(cpes::launch_probe_copy(src_dev, dst_dev, bytes, nontemporal != 0, (hipStream_t)stream), fn);
}

int cpes_rng_probe(uint64_t seed, int64_t n, uint32_t* sink_dev, void* stream)
{
    g_error.clear();
    if (!sink_dev || n < 0) return fail(CPES_ERR_INVALID_ARGUMENT, "cpes_rng_probe: bad sink or count");
    return hip_status(cpes::launch_rng_probe(seed, n, sink_dev, (hipStream_t)stream), "cpes_rng_probe");
}

}  // extern "C"
