// cpes_kernels.hip -- gfx950 kernels of the CoPES parameter-space hot path.
//
// Streaming kernels (perturb, restore, master staging, update) work on
// "units" of consecutive subspace positions: 8 for bf16 weights (one 16-byte
// vector, two Philox blocks) and 4 for fp32 weights (one 16-byte vector, one
// Philox block), one unit per thread at a time.  A wave therefore moves 1 KiB
// per vector access, fully coalesced.  Units whose 16-byte vectors are not
// aligned (an odd subspace offset, an odd map entry) and the ragged tail take
// an element-by-element path with the same arithmetic.  Subspaces are ranges,
// int64 or uint32 element maps, or chunk lists.  Noise never leaves registers.
#include <algorithm>
#include <type_traits>

#include "cpes_device.hpp"
#include "cpes_launch.hpp"

namespace cpes {

namespace {

template <typename T> struct UnitOf;
template <> struct UnitOf<uint16_t> { static constexpr int n = 8; };
template <> struct UnitOf<float> { static constexpr int n = 4; };

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf16_to_f32(v); }
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) { return f32_to_bf16(v); }
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }

template <int N>
__device__ __forceinline__ void unit_normals(uint32_t k0, uint32_t k1, uint64_t q, const BmTables* tb, float z[N]);
template <>
__device__ __forceinline__ void unit_normals<4>(uint32_t k0, uint32_t k1, uint64_t q, const BmTables* tb, float z[4])
{
    normals4(k0, k1, q, tb, z);
}
template <>
__device__ __forceinline__ void unit_normals<8>(uint32_t k0, uint32_t k1, uint64_t q, const BmTables* tb, float z[8])
{
    normals8(k0, k1, q, tb, z);
}

// 16-byte vector loads / stores of one unit.  NT marks the accesses
// non-temporal: a copy far larger than the caches (a subspace of 10^8
// parameters and up) then streams past them instead of evicting lines that
// are never reused, which measured 3-5 % faster on such copies; copies of a
// few tens of MB keep the default policy, since they run from cache.
typedef unsigned int V4u __attribute__((ext_vector_type(4)));
typedef float V4f __attribute__((ext_vector_type(4)));

template <typename T, bool NT = false>
__device__ __forceinline__ void load_vec(const T* p, T v[UnitOf<T>::n])
{
    const V4u* q = reinterpret_cast<const V4u*>(p);
    *reinterpret_cast<V4u*>(v) = NT ? __builtin_nontemporal_load(q) : *q;
}
template <typename T, bool NT = false>
__device__ __forceinline__ void store_vec(T* p, const T v[UnitOf<T>::n])
{
    const V4u x = *reinterpret_cast<const V4u*>(v);
    if (NT)
        __builtin_nontemporal_store(x, reinterpret_cast<V4u*>(p));
    else
        *reinterpret_cast<V4u*>(p) = x;
}
template <int N, bool NT = false>
__device__ __forceinline__ void load_f32s(const float* p, float v[N])
{
#pragma unroll
    for (int h = 0; h < N / 4; ++h) {
        const V4f* q = reinterpret_cast<const V4f*>(p) + h;
        const V4f x = NT ? __builtin_nontemporal_load(q) : *q;
        v[4 * h + 0] = x[0]; v[4 * h + 1] = x[1]; v[4 * h + 2] = x[2]; v[4 * h + 3] = x[3];
    }
}
template <int N, bool NT = false>
__device__ __forceinline__ void store_f32s(float* p, const float v[N])
{
#pragma unroll
    for (int h = 0; h < N / 4; ++h) {
        const V4f x = {v[4 * h + 0], v[4 * h + 1], v[4 * h + 2], v[4 * h + 3]};
        if (NT)
            __builtin_nontemporal_store(x, reinterpret_cast<V4f*>(p) + h);
        else
            reinterpret_cast<V4f*>(p)[h] = x;
    }
}
__device__ __forceinline__ int64_t grid_stride() { return (int64_t)gridDim.x * blockDim.x; }
__device__ __forceinline__ int64_t global_tid() { return (int64_t)blockIdx.x * blockDim.x + threadIdx.x; }

// Subspace addressing: position j is parameter offset + j (kContig),
// index[offset + j] (kGather), or, with chunks of 2^s parameters,
// index[offset + (j >> s)] * 2^s + (j mod 2^s) (kChunk).
constexpr int kContig = kAddrContig, kGather = kAddrGather, kChunk = kAddrChunk, kGather32 = kAddrGather32;

// An element-level map (int64 or uint32 entries).
template <int ADDR>
constexpr bool kMap = ADDR == kGather || ADDR == kGather32;

// Resolve the parameter index of position j; returns false for a map entry
// outside [0, numel) (skipped, never dereferenced).
template <int ADDR>
__device__ __forceinline__ bool param_at(const int64_t* index, int64_t offset, int64_t numel, int shift, int64_t j,
                                         int64_t& i)
{
    if (ADDR == kContig) {
        i = offset + j;
        return true;
    }
    if (ADDR == kGather) {
        i = index[offset + j];
        return i >= 0 && i < numel;
    }
    if (ADDR == kGather32) {
        i = reinterpret_cast<const uint32_t*>(index)[offset + j];
        return i < numel;
    }
    const int64_t c = index[offset + (j >> shift)];
    if (c < 0 || c > (numel >> shift)) return false;
    i = (c << shift) + (j & ((1ll << shift) - 1));
    return i < numel;
}

template <int ADDR>
__device__ __forceinline__ bool param_of(const StreamArgs& a, int64_t j, int64_t& i)
{
    return param_at<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j, i);
}

// First parameter of the unit starting at position j0 for contiguous and
// chunked subspaces (a unit never crosses a chunk); false if the unit would
// leave [0, numel), in which case the caller takes the element path.
//
// The 64 lanes of a wave always hold 64 consecutive units whose first
// position is a multiple of 64 n.  When a chunk holds at least 64 n positions
// the whole wave therefore lies in one chunk, and its chunk id is read once,
// by a scalar load from the wave's first active lane: the chunk list is
// read-only here, so it is addressed as constant memory.
typedef const int64_t __attribute__((address_space(4)))* ConstI64;

__device__ __forceinline__ int64_t wave_uniform(int64_t x)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

template <int ADDR>
__device__ __forceinline__ bool unit_base(const int64_t* index, int64_t offset, int64_t numel, int shift, int64_t j0,
                                          int n, int64_t& base)
{
    if (ADDR == kContig) {
        base = offset + j0;
        return true;
    }
    int64_t c;
    if ((int64_t)64 * n <= (1ll << shift))
        c = ((ConstI64)(uintptr_t)index)[offset + (wave_uniform(j0) >> shift)];
    else
        c = index[offset + (j0 >> shift)];
    if (c < 0 || c > (numel >> shift)) return false;
    base = (c << shift) + (j0 & ((1ll << shift) - 1));
    return base + n <= numel;
}

// Drive a streaming kernel: every full unit goes through `vec_body` (16-byte
// accesses; only when the subspace's vectors are aligned) or `scalar_body`
// (element accesses) in a branch-free grid-stride loop, so that per-launch
// invariants (polynomial constants, key schedule) stay hoisted; the ragged
// last unit, if any, is done once by thread 0 with `scalar_body`.
template <int N, bool VEC, typename VecBody, typename ScalarBody>
__device__ __forceinline__ void for_each_unit(int64_t length, VecBody&& vec_body, ScalarBody&& scalar_body)
{
    const int64_t full = length / N;
    if (VEC) {
        for (int64_t u = global_tid(); u < full; u += grid_stride()) vec_body(u);
    } else {
        for (int64_t u = global_tid(); u < full; u += grid_stride()) scalar_body(u);
    }
    if (full * N < length && global_tid() == 0) scalar_body(full);
}

// ---------------------------------------------------------------- perturb --
// w[p(j)] = cast(fmaf(scale, eps_j, src_j)); src = w (optionally backed up to
// the snapshot first), the fp32 master, or an existing backup.  Also serves
// replay restore with scale = -sign * sigma.  Contiguous and chunked
// subspaces; index maps take k_perturb_map below.
template <typename T, int AUX, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_perturb(StreamArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    T* w = static_cast<T*>(a.w);
    auto scalar_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        float z[N];
        unit_normals<N>(a.k0, a.k1, (uint64_t)(a.noise0 + j0) >> 2, tb, z);
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = j0 + e;
            int64_t i;
            if (j >= a.length || !param_of<ADDR>(a, j, i)) continue;
            float src;
            if (AUX == kAuxMaster) {
                src = static_cast<const float*>(a.aux)[j];
            } else if (AUX == kAuxBackup) {
                src = to_f32<T>(static_cast<const T*>(a.aux)[j]);
            } else {
                const T old = w[i];
                if (AUX == kAuxSnapshot) static_cast<T*>(a.aux)[j] = old;
                src = to_f32<T>(old);
            }
            w[i] = from_f32<T>(__builtin_fmaf(a.scale, z[e], src));
        }
    };
    auto vec_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        int64_t base = 0;
        if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_body(u);
            return;
        }
        float src[N];
        T old[N];
        if (AUX != kAuxMaster && AUX != kAuxBackup) load_vec<T>(w + base, old);
        if (AUX == kAuxMaster) {
            load_f32s<N>(static_cast<const float*>(a.aux) + j0, src);
        } else if (AUX == kAuxBackup) {
            T b[N];
            load_vec<T>(static_cast<const T*>(a.aux) + j0, b);
#pragma unroll
            for (int e = 0; e < N; ++e) src[e] = to_f32<T>(b[e]);
        } else {
#pragma unroll
            for (int e = 0; e < N; ++e) src[e] = to_f32<T>(old[e]);
            if (AUX == kAuxSnapshot) store_vec<T>(static_cast<T*>(a.aux) + j0, old);
        }
        float z[N];
        unit_normals<N>(a.k0, a.k1, (uint64_t)(a.noise0 + j0) >> 2, tb, z);
        T out[N];
#pragma unroll
        for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(a.scale, z[e], src[e]));
        store_vec<T>(w + base, out);
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// --------------------------------------------------------------- restores --
// Snapshot restore: w[p(j)] = snap[j], a bit copy.
template <typename T, bool NT, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_restore_copy(StreamArgs a)
{
    constexpr int N = UnitOf<T>::n;
    T* w = static_cast<T*>(a.w);
    const T* snap = static_cast<const T*>(a.aux);
    auto scalar_body = [&](int64_t u) {
        const int64_t j0 = u * N;
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = j0 + e;
            int64_t i;
            if (j < a.length && param_of<ADDR>(a, j, i)) w[i] = snap[j];
        }
    };
    auto vec_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        int64_t base;
        if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_body(u);
            return;
        }
        T v[N];
        load_vec<T, NT>(snap + j0, v);
        store_vec<T, NT>(w + base, v);
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// Backup copy: backup[j] = w[p(j)] (bit copy), for backups taken apart from a
// perturbation, in device memory or in pinned host memory.
template <typename T, bool NT, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_backup_copy(StreamArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const T* w = static_cast<const T*>(a.w);
    T* backup = static_cast<T*>(a.aux);
    auto scalar_body = [&](int64_t u) {
        const int64_t j0 = u * N;
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = j0 + e;
            int64_t i;
            if (j < a.length) backup[j] = param_of<ADDR>(a, j, i) ? w[i] : T(0);
        }
    };
    auto vec_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        int64_t base;
        if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_body(u);
            return;
        }
        T v[N];
        load_vec<T, NT>(w + base, v);
        store_vec<T, NT>(backup + j0, v);
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// Master restore (bf16 weights): w[p(j)] = rne_bf16(master[j]).
template <bool NT, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_restore_master(StreamArgs a)
{
    constexpr int N = 8;
    uint16_t* w = static_cast<uint16_t*>(a.w);
    const float* master = static_cast<const float*>(a.aux);
    auto scalar_body = [&](int64_t u) {
        const int64_t j0 = u * N;
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = j0 + e;
            int64_t i;
            if (j < a.length && param_of<ADDR>(a, j, i)) w[i] = f32_to_bf16(master[j]);
        }
    };
    auto vec_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        int64_t base;
        if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_body(u);
            return;
        }
        float m[N];
        load_f32s<N, NT>(master + j0, m);
        uint16_t v[N];
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = f32_to_bf16(m[e]);
        store_vec<uint16_t, NT>(w + base, v);
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// Master staging: master[j] = f32(w[p(j)]).
template <typename T, bool NT, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_stage_master(StreamArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const T* w = static_cast<const T*>(a.w);
    float* master = static_cast<float*>(a.aux);
    auto scalar_body = [&](int64_t u) {
        const int64_t j0 = u * N;
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = j0 + e;
            int64_t i;
            if (j < a.length && param_of<ADDR>(a, j, i)) master[j] = to_f32<T>(w[i]);
        }
    };
    auto vec_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        int64_t base;
        if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_body(u);
            return;
        }
        T v[N];
        load_vec<T, NT>(w + base, v);
        float m[N];
#pragma unroll
        for (int e = 0; e < N; ++e) m[e] = to_f32<T>(v[e]);
        store_f32s<N, NT>(master + j0, m);
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// ----------------------------------------------------------------- update --
// theta_S += step * sum_u c_u eps_u, c_u = sum over members of stream u of
// sign * rnorm.  Each thread reads its unit of weights once, regenerates every
// stream's noise for it in registers, accumulates in fp32 and writes once.

// Fold members into stream coefficients, in member order, in fp64.
__device__ __forceinline__ void fold_coefficients(const int32_t n_members, const int32_t n_streams,
                                                  const uint8_t* member_stream, const int8_t* member_sign,
                                                  const float* rnorm, float* coef)
{
    for (int u = threadIdx.x; u < n_streams; u += blockDim.x) {
        double c = 0.0;
        for (int i = 0; i < n_members; ++i)
            if (member_stream[i] == u) c += (double)member_sign[i] * (double)rnorm[i];
        coef[u] = (float)c;
    }
    __syncthreads();
}

// acc[e] = sum over streams s0 <= s < s1 of coef[s] * eps_s(q-th block pair), in stream order.
template <int N>
__device__ __forceinline__ void accumulate_streams(const uint32_t* seed_lo, const uint32_t* seed_hi, const float* coef,
                                                   int s0, int s1, uint64_t q, const BmTables* tb, float acc[N])
{
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = 0.0f;
    for (int s = s0; s < s1; ++s) {
        const float c = coef[s];
        float z[N];
        unit_normals<N>(seed_lo[s], seed_hi[s], q, tb, z);
#pragma unroll
        for (int e = 0; e < N; ++e) acc[e] = __builtin_fmaf(c, z[e], acc[e]);
    }
}

template <typename T, bool MASTER, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_update(UpdateArgs a)
{
    constexpr int N = MASTER ? 8 : UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    __shared__ float coef[kMaxMembers];
    fold_coefficients(a.n_members, a.n_streams, a.member_stream, a.member_sign, a.rnorm, coef);

    T* w = static_cast<T*>(a.w);
    auto accumulate = [&](int64_t j0, float acc[N]) {
        accumulate_streams<N>(a.seed_lo, a.seed_hi, coef, 0, a.n_streams, (uint64_t)(a.noise0 + j0) >> 2, tb, acc);
    };
    auto scalar_finish = [&](int64_t j0, const float acc[N]) {
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = j0 + e;
            int64_t i;
            if (j >= a.length || !param_at<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j, i)) continue;
            if (MASTER) {
                const float m = __builtin_fmaf(a.step, acc[e], a.master[j]);
                a.master[j] = m;
                w[i] = from_f32<T>(m);
            } else {
                w[i] = from_f32<T>(__builtin_fmaf(a.step, acc[e], to_f32<T>(w[i])));
            }
        }
    };
    auto scalar_body = [&](int64_t u) {
        float acc[N];
        accumulate(u * N, acc);
        scalar_finish(u * N, acc);
    };
    auto vec_body = [&](int64_t u) {
        const int64_t j0 = u * N;
        float acc[N];
        accumulate(j0, acc);
        int64_t base = 0;
        T v[N];
        if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_finish(j0, acc);
            return;
        }
        if (!MASTER) load_vec<T>(w + base, v);
        T out[N];
        if (MASTER) {
            float m[N];
            load_f32s<N>(a.master + j0, m);
#pragma unroll
            for (int e = 0; e < N; ++e) {
                m[e] = __builtin_fmaf(a.step, acc[e], m[e]);
                out[e] = from_f32<T>(m[e]);
            }
            store_f32s<N>(a.master + j0, m);
        } else {
#pragma unroll
            for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(a.step, acc[e], to_f32<T>(v[e])));
        }
        store_vec<T>(w + base, out);
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// ------------------------------------------------------- index-map kernels --
// Subspaces given by an element map (int64 or uint32 entries; a partition's
// maps are ascending, at density d_k / d across the weights).  A wave owns
// tiles of 64 N consecutive positions.  Map entries, and the weights they
// address, are taken lane-interleaved: lane l handles positions t0 + l + 64 e,
// e < N.  Each memory instruction then covers 64 consecutive map entries, a
// window of about 64 d / d_k consecutive weights (a few 128-byte lines), where
// a unit per lane would touch 64 windows that far apart.  Noise comes in
// units of N consecutive positions per lane, and so do contiguous side
// buffers (backup, master); a per-wave LDS buffer of one tile converts
// between the two layouts.

template <int ADDR>
__device__ __forceinline__ int64_t map_entry(const int64_t* index, int64_t p)
{
    if (ADDR == kGather) return index[p];
    return (int64_t)reinterpret_cast<const uint32_t*>(index)[p];
}

// The wave's index and the number of waves in the grid (uniform in a wave).
__device__ __forceinline__ int64_t wave_id()
{
    return (int64_t)blockIdx.x * (kBlock / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
}
__device__ __forceinline__ int64_t wave_count() { return (int64_t)gridDim.x * (kBlock / 64); }

// Parameters of lane `lane`'s positions in the tile at t0:
// idx[e] = map[offset + t0 + lane + 64 e], or -1 beyond the subspace or for
// an entry outside [0, numel) (skipped, never dereferenced).  Returns true
// when every entry of the wave is valid (a full tile of a partition's map).
template <int ADDR, int N>
__device__ __forceinline__ bool tile_entries(const int64_t* index, int64_t offset, int64_t length, int64_t numel,
                                             int64_t t0, int lane, int64_t idx[N])
{
    bool ok = true;
    if (t0 + 64 * N <= length) {
#pragma unroll
        for (int e = 0; e < N; ++e) idx[e] = map_entry<ADDR>(index, offset + t0 + lane + 64 * e);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) {
            const int64_t j = t0 + lane + 64 * e;
            idx[e] = j < length ? map_entry<ADDR>(index, offset + j) : -1;
        }
        ok = false;
    }
#pragma unroll
    for (int e = 0; e < N; ++e)
        if ((uint64_t)idx[e] >= (uint64_t)numel) {
            idx[e] = -1;
            ok = false;
        }
    return __builtin_amdgcn_ballot_w64(!ok) == 0;
}

// Gather w at the tile's entries (lane-interleaved); skipped entries read 0.
template <typename T, int N>
__device__ __forceinline__ void gather_lanes(const T* w, const int64_t idx[N], bool all_valid, T v[N])
{
    if (all_valid) {
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = w[idx[e]];
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = idx[e] >= 0 ? w[idx[e]] : T(0);
    }
}

// Scatter lane-interleaved values.  With every entry valid the stores carry
// no branch and issue back to back; a branch around each store would make the
// compiler wait for the loaded data before every one of them.
template <typename T, int N>
__device__ __forceinline__ void scatter_lanes(T* w, const int64_t idx[N], bool all_valid, const T v[N])
{
    if (all_valid) {
#pragma unroll
        for (int e = 0; e < N; ++e) w[idx[e]] = v[e];
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e)
            if (idx[e] >= 0) w[idx[e]] = v[e];
    }
}

// Lane-level ordering of the exchange buffer: LDS accesses of one wave take
// effect in program order, so the compiler only has to keep them in order.
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Units (lane l holds positions N l .. N l + N - 1 of the tile) to lanes
// (lane l holds l + 64 e), and back, through the wave's tile buffer `buf`
// (64 N elements, 16-byte aligned).
template <int BYTES> struct UnitVec;
template <> struct UnitVec<16> { typedef V4u type; };
template <> struct UnitVec<8> { typedef uint2 type; };

template <typename T, int N>
__device__ __forceinline__ void units_to_lanes(T* buf, int lane, const T in[N], T out[N])
{
    typedef typename UnitVec<N * sizeof(T)>::type U;
    *reinterpret_cast<U*>(buf + N * lane) = *reinterpret_cast<const U*>(in);
    wave_lds_sync();
#pragma unroll
    for (int e = 0; e < N; ++e) out[e] = buf[lane + 64 * e];
    wave_lds_sync();
}
template <typename T, int N>
__device__ __forceinline__ void lanes_to_units(T* buf, int lane, const T in[N], T out[N])
{
    typedef typename UnitVec<N * sizeof(T)>::type U;
#pragma unroll
    for (int e = 0; e < N; ++e) buf[lane + 64 * e] = in[e];
    wave_lds_sync();
    *reinterpret_cast<U*>(out) = *reinterpret_cast<const U*>(buf + N * lane);
    wave_lds_sync();
}

// Unit-wise side buffer access at positions j0 .. j0 + N - 1, bounded by
// `length` (a tile may end inside a unit); 16-byte vectors when VEC and the
// unit is whole.
template <typename T, bool VEC, int N>
__device__ __forceinline__ void load_unit(const T* p, int64_t j0, int64_t length, T v[N])
{
    if (VEC && j0 + N <= length) {
        if (sizeof(T) * N == 16) {
            load_vec<T>(p + j0, v);
        } else {
            load_f32s<N>(reinterpret_cast<const float*>(p) + j0, reinterpret_cast<float*>(v));
        }
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = j0 + e < length ? p[j0 + e] : T(0);
    }
}
template <typename T, bool VEC, int N>
__device__ __forceinline__ void store_unit(T* p, int64_t j0, int64_t length, const T v[N])
{
    if (VEC && j0 + N <= length) {
        if (sizeof(T) * N == 16) {
            store_vec<T>(p + j0, v);
        } else {
            store_f32s<N>(reinterpret_cast<float*>(p) + j0, reinterpret_cast<const float*>(v));
        }
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e)
            if (j0 + e < length) p[j0 + e] = v[e];
    }
}

// Perturbation through a map (see k_perturb for the arithmetic).
template <typename T, int AUX, bool VEC, int ADDR>
__global__ __launch_bounds__(kBlock) void k_perturb_map(StreamArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    __shared__ __attribute__((aligned(16))) T xch[kBlock / 64][64 * N];
    const int lane = threadIdx.x & 63;
    T* buf = xch[threadIdx.x / 64];
    T* w = static_cast<T*>(a.w);
    const int64_t tiles = (a.length + 64 * N - 1) / (64 * N);
    for (int64_t t = wave_id(); t < tiles; t += wave_count()) {
        const int64_t t0 = t * 64 * N, j0 = t0 + (int64_t)N * lane;
        int64_t idx[N];
        const bool all_valid = tile_entries<ADDR, N>(a.index, a.offset, a.length, a.numel, t0, lane, idx);
        float src[N];
        if (AUX == kAuxMaster) {
            load_unit<float, VEC, N>(static_cast<const float*>(a.aux), j0, a.length, src);
        } else {
            T old[N];
            if (AUX == kAuxBackup) {
                load_unit<T, VEC, N>(static_cast<const T*>(a.aux), j0, a.length, old);
            } else {
                T g[N];
                gather_lanes<T, N>(w, idx, all_valid, g);
                lanes_to_units<T, N>(buf, lane, g, old);
                if (AUX == kAuxSnapshot) store_unit<T, VEC, N>(static_cast<T*>(a.aux), j0, a.length, old);
            }
#pragma unroll
            for (int e = 0; e < N; ++e) src[e] = to_f32<T>(old[e]);
        }
        float z[N];
        unit_normals<N>(a.k0, a.k1, (uint64_t)(a.noise0 + j0) >> 2, tb, z);
        T out[N], v[N];
#pragma unroll
        for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(a.scale, z[e], src[e]));
        units_to_lanes<T, N>(buf, lane, out, v);
        scatter_lanes<T, N>(w, idx, all_valid, v);
    }
}

// Copies through a map, all lane-interleaved (no noise, no exchange):
// KIND 0: w[p(j)] = aux[j] (restore from the backup);
// KIND 1: aux[j] = w[p(j)] (backup; skipped entries give 0);
// KIND 2: w[p(j)] = rne_bf16(master[j]) (restore from a master);
// KIND 3: master[j] = f32(w[p(j)]) (master staging).
constexpr int kCopyRestore = 0, kCopyBackup = 1, kCopyRestoreMaster = 2, kCopyStageMaster = 3;

template <typename T, int KIND, bool NT, int ADDR>
__global__ __launch_bounds__(kBlock) void k_copy_map(StreamArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const int lane = threadIdx.x & 63;
    T* w = static_cast<T*>(a.w);
    const int64_t tiles = (a.length + 64 * N - 1) / (64 * N);
    for (int64_t t = wave_id(); t < tiles; t += wave_count()) {
        const int64_t t0 = t * 64 * N;
        int64_t idx[N];
        const bool all_valid = tile_entries<ADDR, N>(a.index, a.offset, a.length, a.numel, t0, lane, idx);
        const bool full = t0 + 64 * N <= a.length;
        if (KIND == kCopyRestore || KIND == kCopyRestoreMaster) {
            T v[N];
#pragma unroll
            for (int e = 0; e < N; ++e) {
                const int64_t j = t0 + lane + 64 * e;
                if (KIND == kCopyRestore) {
                    const T* snap = static_cast<const T*>(a.aux);
                    v[e] = full || j < a.length ? (NT ? __builtin_nontemporal_load(snap + j) : snap[j]) : T(0);
                } else {
                    const float* master = static_cast<const float*>(a.aux);
                    const float m = full || j < a.length ? (NT ? __builtin_nontemporal_load(master + j) : master[j])
                                                        : 0.0f;
                    v[e] = from_f32<T>(m);
                }
            }
            scatter_lanes<T, N>(w, idx, all_valid, v);
        } else {
            T v[N];
            gather_lanes<T, N>(w, idx, all_valid, v);
#pragma unroll
            for (int e = 0; e < N; ++e) {
                const int64_t j = t0 + lane + 64 * e;
                if (!full && j >= a.length) continue;
                if (KIND == kCopyBackup) {
                    T* backup = static_cast<T*>(a.aux);
                    if (NT) __builtin_nontemporal_store(v[e], backup + j);
                    else backup[j] = v[e];
                } else {
                    float* master = static_cast<float*>(a.aux);
                    if (NT) __builtin_nontemporal_store(to_f32<T>(v[e]), master + j);
                    else master[j] = to_f32<T>(v[e]);
                }
            }
        }
    }
}

// ------------------------------------------ dense windows on ascending maps --
// Restores through a strictly ascending element map (a partition's own maps,
// flagged CPES_SUB_ASCENDING).  The weights a wave tile of kDenseTile entries
// touches lie in a narrow window of 128-byte lines.  Each line belongs to the
// tile holding the line's first entry of the subspace; that tile's wave reads
// its lines whole into LDS, overlays its entries -- and those of the next
// tile that fall in its last line (at most 63, the "spill") -- and writes the
// lines back whole.  Each line is then written once and in full, where
// scattered 2-byte stores leave a partial write in nearly every 32-byte
// sector at density 1/8, which the memory system completes by reading the
// sector first.  The other parameters in those lines are written back with
// the values just read.  A tile whose lines do not fit the window (a
// subspace sparser than about 1/10) stores its entries one by one, keeping
// line ownership: it still takes its spill and leaves the entries in a shared
// first line to the previous tile.  bf16 weights only; any map entry outside
// [0, numel) is skipped.  (Perturbations tile without a spill, below, so
// that a wave generates the noise of its own tile's positions only.)
constexpr int kDenseTile = 256;      // entries per wave tile: 4 per lane
constexpr int kDensePer = kDenseTile / 64;
constexpr int kLineElems = 64;       // bf16 elements per 128-byte line
constexpr int kDenseLines = 40;      // LDS window per wave: 5 KiB

struct DenseTile {
    int64_t t0, t1;     // the tile's entries [t0, t1)
    int64_t lo, hi;     // lines [lo, hi] it owns
    bool window;        // the owned lines fit the LDS window (and the tile's ends are in range)
};

template <int ADDR>
__device__ __forceinline__ DenseTile dense_tile(const int64_t* index, int64_t offset, int64_t length, int64_t numel,
                                                int64_t t, int64_t tile)
{
    DenseTile d;
    d.t0 = t * tile;
    d.t1 = d.t0 + tile < length ? d.t0 + tile : length;
    const int64_t first = wave_uniform(map_entry<ADDR>(index, offset + d.t0));
    const int64_t last = wave_uniform(map_entry<ADDR>(index, offset + d.t1 - 1));
    const int64_t A = first >> 6, B = last >> 6;      // floor division by kLineElems
    bool shared = false;
    if (d.t0 > 0) shared = (wave_uniform(map_entry<ADDR>(index, offset + d.t0 - 1)) >> 6) == A;
    d.lo = shared ? A + 1 : A;
    d.hi = B;
    d.window = first >= 0 && last < numel && first <= last && d.hi - d.lo + 1 <= kDenseLines;
    return d;
}

// The tile's own entries (lane-interleaved: position t0 + lane + 64 e) with
// the entries of a shared first line dropped, and this lane's spill entry
// (position t1 + lane, kept if it falls in line hi); -1 where there is none.
template <int ADDR>
__device__ __forceinline__ void dense_entries(const int64_t* index, int64_t offset, int64_t length, int64_t numel,
                                              const DenseTile& d, int lane, int64_t idx[kDensePer], int64_t& sidx)
{
#pragma unroll
    for (int e = 0; e < kDensePer; ++e) {
        const int64_t j = d.t0 + lane + 64 * e;
        int64_t i = j < d.t1 ? map_entry<ADDR>(index, offset + j) : -1;
        if ((uint64_t)i >= (uint64_t)numel || (i >> 6) < d.lo) i = -1;
        idx[e] = i;
    }
    sidx = -1;
    const int64_t j = d.t1 + lane;
    if (j < length) {
        const int64_t i = map_entry<ADDR>(index, offset + j);
        if ((uint64_t)i < (uint64_t)numel && (i >> 6) == d.hi) sidx = i;
    }
}

// Window transfers: lines [lo, hi] of w to and from the wave's LDS buffer,
// one 16-byte vector per lane per step, non-temporal (the weights far exceed
// the caches); the element path covers a window running past numel.
__device__ __forceinline__ void window_load(const uint16_t* w, int64_t numel, const DenseTile& d, uint16_t* buf,
                                            int lane)
{
    const int64_t base = d.lo * kLineElems, nvec = (d.hi - d.lo + 1) * (kLineElems / 8);
    const bool whole = base + nvec * 8 <= numel;
    for (int64_t v = lane; v < nvec; v += 64) {
        if (whole) {
            *reinterpret_cast<V4u*>(buf + 8 * v) =
                __builtin_nontemporal_load(reinterpret_cast<const V4u*>(w + base) + v);
        } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int64_t i = base + 8 * v + k;
                buf[8 * v + k] = i < numel ? w[i] : (uint16_t)0;
            }
        }
    }
}
__device__ __forceinline__ void window_store(uint16_t* w, int64_t numel, const DenseTile& d, const uint16_t* buf,
                                             int lane)
{
    const int64_t base = d.lo * kLineElems, nvec = (d.hi - d.lo + 1) * (kLineElems / 8);
    const bool whole = base + nvec * 8 <= numel;
    for (int64_t v = lane; v < nvec; v += 64) {
        if (whole) {
            __builtin_nontemporal_store(*reinterpret_cast<const V4u*>(buf + 8 * v),
                                        reinterpret_cast<V4u*>(w + base) + v);
        } else {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int64_t i = base + 8 * v + k;
                if (i < numel) w[i] = buf[8 * v + k];
            }
        }
    }
}

// Write the tile's new values: overlaid on the window and stored whole, or
// (no window) stored one by one.
__device__ __forceinline__ void dense_write(uint16_t* w, int64_t numel, const DenseTile& d, uint16_t* buf, int lane,
                                            const int64_t idx[kDensePer], const uint16_t v[kDensePer], int64_t sidx,
                                            uint16_t sv)
{
    if (d.window) {
        const int64_t base = d.lo * kLineElems, nelem = (d.hi - d.lo + 1) * kLineElems;
#pragma unroll
        for (int e = 0; e < kDensePer; ++e)
            if (idx[e] >= base && idx[e] < base + nelem) buf[idx[e] - base] = v[e];
        if (sidx >= base && sidx < base + nelem) buf[sidx - base] = sv;
        wave_lds_sync();
        window_store(w, numel, d, buf, lane);
        wave_lds_sync();
    } else {
#pragma unroll
        for (int e = 0; e < kDensePer; ++e)
            if (idx[e] >= 0) w[idx[e]] = v[e];
        if (sidx >= 0) w[sidx] = sv;
    }
}

// Restore through an ascending map: w[p(j)] = aux[j] (bf16 backup, KIND
// kCopyRestore) or rne_bf16(aux[j]) (fp32 master, KIND kCopyRestoreMaster).
template <int KIND, int ADDR>
__global__ __launch_bounds__(kBlock) void k_restore_dense(StreamArgs a)
{
    __shared__ __attribute__((aligned(16))) uint16_t win[kBlock / 64][kDenseLines * kLineElems];
    const int lane = threadIdx.x & 63;
    uint16_t* buf = win[threadIdx.x / 64];
    uint16_t* w = static_cast<uint16_t*>(a.w);
    auto source = [&](int64_t j) -> uint16_t {
        if (KIND == kCopyRestore) return __builtin_nontemporal_load(static_cast<const uint16_t*>(a.aux) + j);
        return f32_to_bf16(__builtin_nontemporal_load(static_cast<const float*>(a.aux) + j));
    };
    const int64_t tiles = (a.length + kDenseTile - 1) / kDenseTile;
    for (int64_t t = wave_id(); t < tiles; t += wave_count()) {
        const DenseTile d = dense_tile<ADDR>(a.index, a.offset, a.length, a.numel, t, kDenseTile);
        int64_t idx[kDensePer], sidx;
        dense_entries<ADDR>(a.index, a.offset, a.length, a.numel, d, lane, idx, sidx);
        uint16_t v[kDensePer], sv = 0;
#pragma unroll
        for (int e = 0; e < kDensePer; ++e) v[e] = idx[e] >= 0 ? source(d.t0 + lane + 64 * e) : (uint16_t)0;
        if (sidx >= 0) sv = source(d.t1 + lane);
        if (d.window) {
            window_load(w, a.numel, d, buf, lane);
            wave_lds_sync();
        }
        dense_write(w, a.numel, d, buf, lane, idx, v, sidx, sv);
    }
}

// ----------------------------------- whole-line perturbations (ascending) --
// A perturbation through an ascending map writes whole lines too, on fixed
// tiles of kDenseTile entries but without a spill: the lines strictly inside
// a tile's span hold no entry of another tile and go through the tile's LDS
// window; its entries in a first or last line shared with a neighbouring tile
// are stored one by one, as the neighbour stores its own entries there, so a
// line written whole has no other writer.  Lane l takes the tile's positions
// t0 + 4 l .. t0 + 4 l + 3, which are one Philox block of noise, and moves
// the map and the side buffers as 8- or 16-byte vectors where aligned.  The
// perturbation is that of Eq. (8) on a subspace of the partition of Eq. (7).
// (Restores tiled this way, with no noise to generate, measured a few per
// cent slower than the spill kernel above, which they therefore keep.)
template <int ADDR>
__device__ __forceinline__ DenseTile edge_tile(const int64_t* index, int64_t offset, int64_t length, int64_t numel,
                                               int64_t t)
{
    DenseTile d;
    d.t0 = t * kDenseTile;
    d.t1 = d.t0 + kDenseTile < length ? d.t0 + kDenseTile : length;
    const int64_t first = wave_uniform(map_entry<ADDR>(index, offset + d.t0));
    const int64_t last = wave_uniform(map_entry<ADDR>(index, offset + d.t1 - 1));
    const int64_t A = first >> 6, B = last >> 6;
    const bool prev = d.t0 > 0 && (wave_uniform(map_entry<ADDR>(index, offset + d.t0 - 1)) >> 6) == A;
    const bool next = d.t1 < length && (wave_uniform(map_entry<ADDR>(index, offset + d.t1)) >> 6) == B;
    d.lo = prev ? A + 1 : A;
    d.hi = next ? B - 1 : B;
    if (d.hi < d.lo) d.hi = d.lo - 1;   // every entry lies in a shared line: an empty window
    d.window = first >= 0 && last < numel && first <= last && d.hi - d.lo + 1 <= kDenseLines;
    return d;
}

// Entries p .. p + 3 of the map (n of them exist; -1 for the others and for
// entries outside [0, numel)); vector loads when `vec` (16-byte aligned).
template <int ADDR>
__device__ __forceinline__ void map_entries4(const int64_t* index, int64_t p, int64_t n, bool vec, int64_t numel,
                                             int64_t idx[4])
{
    if (vec && n >= 4) {
        if (ADDR == kGather) {
            const V4u x = *reinterpret_cast<const V4u*>(index + p);
            const V4u y = *reinterpret_cast<const V4u*>(index + p + 2);
            idx[0] = (int64_t)(((uint64_t)x[1] << 32) | x[0]);
            idx[1] = (int64_t)(((uint64_t)x[3] << 32) | x[2]);
            idx[2] = (int64_t)(((uint64_t)y[1] << 32) | y[0]);
            idx[3] = (int64_t)(((uint64_t)y[3] << 32) | y[2]);
        } else {
            const V4u x = *reinterpret_cast<const V4u*>(reinterpret_cast<const uint32_t*>(index) + p);
#pragma unroll
            for (int e = 0; e < 4; ++e) idx[e] = (int64_t)x[e];
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) idx[e] = e < n ? map_entry<ADDR>(index, p + e) : -1;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if ((uint64_t)idx[e] >= (uint64_t)numel) idx[e] = -1;
}

// The tile's new values: those in the window (in[e]) overlaid on it and its
// lines stored whole, the others (in a shared line, or all of them when the
// tile has no window) stored one by one.
__device__ __forceinline__ void edge_write(uint16_t* w, int64_t numel, const DenseTile& d, uint16_t* buf, int lane,
                                           const int64_t idx[4], const bool in[4], int64_t base, const uint16_t v[4])
{
    if (d.window) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (in[e]) buf[idx[e] - base] = v[e];
        wave_lds_sync();
        window_store(w, numel, d, buf, lane);
        wave_lds_sync();
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (!in[e] && idx[e] >= 0) w[idx[e]] = v[e];
}

// Workgroups of kDenseBlock threads share one copy of the noise tables; with
// at most 80 VGPRs, three of them (52 KiB of LDS each) give 6 waves per SIMD,
// where 256-thread workgroups (32 KiB each) give 5.  Measured on 0.5 G-entry
// maps: 6-20 % faster, except the perturbation from the backup through an
// int64 map (3 % slower).
constexpr int kDenseBlock = 512;

template <int AUX, int ADDR>
__global__ __launch_bounds__(kDenseBlock, 6) void k_perturb_dense(StreamArgs a)
{
    const BmTables* tb = stage_bm_tables<kDenseBlock>();
    __shared__ __attribute__((aligned(16))) uint16_t win[kDenseBlock / 64][kDenseLines * kLineElems];
    const int lane = threadIdx.x & 63;
    uint16_t* buf = win[threadIdx.x / 64];
    uint16_t* w = static_cast<uint16_t*>(a.w);
    constexpr uint64_t kEntry = ADDR == kGather ? 8 : 4;
    const bool vmap = (((uintptr_t)a.index + (uint64_t)a.offset * kEntry) & 15) == 0;
    const bool vaux = ((uintptr_t)a.aux & (AUX == kAuxMaster ? 15 : 7)) == 0;
    const int64_t tiles = (a.length + kDenseTile - 1) / kDenseTile;
    const int64_t waves = (int64_t)gridDim.x * (kDenseBlock / 64);
    for (int64_t t = (int64_t)blockIdx.x * (kDenseBlock / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x / 64); t < tiles;
         t += waves) {
        const DenseTile d = edge_tile<ADDR>(a.index, a.offset, a.length, a.numel, t);
        const int64_t j0 = d.t0 + 4 * lane;
        const bool whole = j0 + 4 <= a.length;
        int64_t idx[4];
        map_entries4<ADDR>(a.index, a.offset + j0, a.length - j0, vmap, a.numel, idx);
        float src[4];
        if (AUX == kAuxBackup) {
            const uint16_t* b = static_cast<const uint16_t*>(a.aux) + j0;
            uint16_t o[4];
            if (vaux && whole) {
                *reinterpret_cast<uint2*>(o) = *reinterpret_cast<const uint2*>(b);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = j0 + e < a.length ? b[e] : (uint16_t)0;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) src[e] = bf16_to_f32(o[e]);
        } else if (AUX == kAuxMaster) {
            const float* m = static_cast<const float*>(a.aux) + j0;
            if (vaux && whole) {
                load_f32s<4>(m, src);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) src[e] = j0 + e < a.length ? m[e] : 0.0f;
            }
        }
        float z[4];
        normals4(a.k0, a.k1, (uint64_t)(a.noise0 + j0) >> 2, tb, z);
        int64_t base = 0, nelem = 0;
        if (d.window) {
            base = d.lo * kLineElems;
            nelem = (d.hi - d.lo + 1) * kLineElems;
            window_load(w, a.numel, d, buf, lane);
            wave_lds_sync();
        }
        bool in[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) in[e] = idx[e] >= base && idx[e] < base + nelem;
        if (AUX == kAuxNone || AUX == kAuxSnapshot) {
            uint16_t o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = in[e] ? buf[idx[e] - base] : idx[e] >= 0 ? w[idx[e]] : (uint16_t)0;
            if (AUX == kAuxSnapshot) {
                uint16_t* snap = static_cast<uint16_t*>(a.aux) + j0;
                if (vaux && whole) {
                    *reinterpret_cast<uint2*>(snap) = *reinterpret_cast<const uint2*>(o);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (j0 + e < a.length) snap[e] = o[e];
                }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) src[e] = bf16_to_f32(o[e]);
        }
        uint16_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = f32_to_bf16(__builtin_fmaf(a.scale, z[e], src[e]));
        edge_write(w, a.numel, d, buf, lane, idx, in, base, v);
    }
}

// Update through a map (see k_update for the arithmetic).
template <typename T, bool MASTER, bool VEC, int ADDR>
__global__ __launch_bounds__(kBlock) void k_update_map(UpdateArgs a)
{
    constexpr int N = UnitOf<T>::n;   // a master update has bf16 weights: N = 8
    const BmTables* tb = stage_bm_tables<kBlock>();
    __shared__ float coef[kMaxMembers];
    __shared__ __attribute__((aligned(16))) T xch[kBlock / 64][64 * N];
    fold_coefficients(a.n_members, a.n_streams, a.member_stream, a.member_sign, a.rnorm, coef);
    const int lane = threadIdx.x & 63;
    T* buf = xch[threadIdx.x / 64];
    T* w = static_cast<T*>(a.w);
    const int64_t tiles = (a.length + 64 * N - 1) / (64 * N);
    for (int64_t t = wave_id(); t < tiles; t += wave_count()) {
        const int64_t t0 = t * 64 * N, j0 = t0 + (int64_t)N * lane;
        int64_t idx[N];
        const bool all_valid = tile_entries<ADDR, N>(a.index, a.offset, a.length, a.numel, t0, lane, idx);
        T g[N];
        if (!MASTER) gather_lanes<T, N>(w, idx, all_valid, g);   // in flight while the noise is generated
        float acc[N];
        accumulate_streams<N>(a.seed_lo, a.seed_hi, coef, 0, a.n_streams, (uint64_t)(a.noise0 + j0) >> 2, tb, acc);
        T out[N], v[N];
        if (MASTER) {
            float m[N];
            load_unit<float, VEC, N>(a.master, j0, a.length, m);
#pragma unroll
            for (int e = 0; e < N; ++e) {
                m[e] = __builtin_fmaf(a.step, acc[e], m[e]);
                out[e] = from_f32<T>(m[e]);
            }
            store_unit<float, VEC, N>(a.master, j0, a.length, m);
        } else {
            T old[N];
            lanes_to_units<T, N>(buf, lane, g, old);
#pragma unroll
            for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(a.step, acc[e], to_f32<T>(old[e])));
        }
        units_to_lanes<T, N>(buf, lane, out, v);
        scatter_lanes<T, N>(w, idx, all_valid, v);
    }
}

// ------------------------------------------------------------ step update --
// theta += sum_k P_k step_k sum_{u in streams of k} c_u eps_u (Eq. 13, Alg. 1):
// every subspace of the partition with its own members, in one launch.  Units
// restart at each subspace's first position, so noise position j is always
// relative to the subspace; each wave works on 64 units of one subspace (one
// tile, taken lane-interleaved on an element map as in the map kernels).
template <typename T, int ADDR>
__global__ __launch_bounds__(kBlock) void k_update_step(StepArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    __shared__ float coef[kMaxMembers];
    __shared__ __attribute__((aligned(16))) T xch[kBlock / 64][64 * N];
    fold_coefficients(a.n_members, a.n_streams, a.member_stream, a.member_sign, a.rnorm, coef);
    T* w = static_cast<T*>(a.w);
    const int lane = threadIdx.x & 63;
    T* buf = xch[threadIdx.x / 64];
    const int64_t tiles = a.tile_begin[a.K];
    for (int64_t t = wave_id(); t < tiles; t += wave_count()) {
        // t is the same for the whole wave; so are k and the stream range, which
        // keeps the seed and coefficient reads scalar
        int k = 0;
        while (k + 1 < a.K && a.tile_begin[k + 1] <= t) ++k;
        k = __builtin_amdgcn_readfirstlane(k);
        const int st0 = __builtin_amdgcn_readfirstlane(a.stream_begin[k]);
        const int st1 = __builtin_amdgcn_readfirstlane(a.stream_begin[k + 1]);
        const int64_t off = a.offset[k];
        const int64_t len = a.length[k];
        const float step = a.step[k];
        const int64_t t0 = (t - a.tile_begin[k]) * 64 * N;
        const int64_t j0 = t0 + (int64_t)N * lane;
        if (kMap<ADDR>) {
            int64_t idx[N];
            const bool all_valid = tile_entries<ADDR, N>(a.index, off, len, a.numel, t0, lane, idx);
            T g[N], old[N], out[N], v[N];
            gather_lanes<T, N>(w, idx, all_valid, g);
            float acc[N];
            accumulate_streams<N>(a.seed_lo, a.seed_hi, coef, st0, st1, (uint64_t)j0 >> 2, tb, acc);
            lanes_to_units<T, N>(buf, lane, g, old);
#pragma unroll
            for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(step, acc[e], to_f32<T>(old[e])));
            units_to_lanes<T, N>(buf, lane, out, v);
            scatter_lanes<T, N>(w, idx, all_valid, v);
            continue;
        }
        if (j0 >= len) continue;
        int64_t base = 0;
        const bool vec = ((a.vec_mask >> k) & 1u) && j0 + N <= len &&
                         unit_base<ADDR>(a.index, off, a.numel, a.chunk_shift, j0, N, base);
        float acc[N];
        accumulate_streams<N>(a.seed_lo, a.seed_hi, coef, st0, st1, (uint64_t)j0 >> 2, tb, acc);
        if (vec) {
            T v[N], out[N];
            load_vec<T>(w + base, v);
#pragma unroll
            for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(step, acc[e], to_f32<T>(v[e])));
            store_vec<T>(w + base, out);
        } else {
#pragma unroll
            for (int e = 0; e < N; ++e) {
                const int64_t j = j0 + e;
                int64_t i;
                if (j >= len || !param_at<ADDR>(a.index, off, a.numel, a.chunk_shift, j, i)) continue;
                w[i] = from_f32<T>(__builtin_fmaf(step, acc[e], to_f32<T>(w[i])));
            }
        }
    }
}

// -------------------------------------------------------------- normalise --
// One workgroup.  The rewards are sorted in LDS by the 64-bit key
// (group, value, index) -- the value as an order-preserving 32-bit image of
// the fp32 bits, -0 taken as +0 -- with a bitonic network.  Each group is
// then one run of the sorted keys, in a canonical order (ascending value).
// Z: one wave per group sums the run in fp64 (lane l takes run entries
// l, l + 64, ... in order, then an xor-shuffle butterfly combines the 64
// partial sums; every lane ends with the same total), for the mean and then
// for the squared deviations.  RANK: the rank of an entry is the start of
// its run of equal values within its group, the number of ties the run's
// length, both found by binary search.
constexpr int kNormThreads = 1024;
constexpr int kNormMaxN = 4096;
constexpr int kNormMaxGroups = 1024;
constexpr int kNormIdxBits = 12;                 // index < kNormMaxN
constexpr int kNormValShift = kNormIdxBits;      // value bits 12 .. 43
constexpr int kNormGroupShift = kNormIdxBits + 32;   // group bits 44 .. 53
static_assert((1 << kNormIdxBits) >= kNormMaxN && kNormMaxGroups <= (1 << (64 - kNormGroupShift - 1)),
              "index, value and group fit the sort key");

__device__ __forceinline__ uint32_t order_bits(float v)
{
    uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_order_bits(uint32_t o)
{
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

// First position p in [0, n) with keys[p] >= x (keys ascending).
__device__ __forceinline__ int lower_bound_u64(const uint64_t* keys, int n, uint64_t x)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (keys[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

__device__ __forceinline__ double wave_sum(double x)
{
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) x += __shfl_xor(x, m, 64);
    return x;
}

__global__ __launch_bounds__(kNormThreads) void k_normalize(NormalizeArgs a)
{
#pragma clang fp contract(off)
    __shared__ uint64_t keys[kNormMaxN];
    __shared__ int32_t start[kNormMaxGroups + 1];
    __shared__ int bad;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    int n2 = 1;
    while (n2 < a.n) n2 <<= 1;
    int my_bad = 0;
    for (int i = threadIdx.x; i < n2; i += blockDim.x) {
        uint64_t key = ~0ull;                              // padding sorts last
        if (i < a.n) {
            const float v = a.r[i];
            const int32_t gi = a.group ? a.group[i] : 0;
            if (!__builtin_isfinite(v)) my_bad |= 1;
            if (gi < 0 || gi >= a.n_groups) my_bad |= 2;
            key = ((uint64_t)(uint32_t)gi << kNormGroupShift) | ((uint64_t)order_bits(v) << kNormValShift) |
                  (uint64_t)i;
        }
        keys[i] = key;
    }
    if (my_bad) atomicOr(&bad, my_bad);
    __syncthreads();
    const int status = (bad & 2) ? 2 : (bad & 1) ? 1 : 0;
    if (status != 0) {
        for (int i = threadIdx.x; i < a.n; i += blockDim.x) a.out[i] = 0.0f;
        if (a.status && threadIdx.x == 0) *a.status = status;
        return;
    }
    // bitonic sort, ascending
    for (int k = 2; k <= n2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < n2; i += blockDim.x) {
                const int p = i ^ j;
                if (p > i) {
                    const uint64_t x = keys[i], y = keys[p];
                    if ((x > y) == ((i & k) == 0)) {
                        keys[i] = y;
                        keys[p] = x;
                    }
                }
            }
            __syncthreads();
        }
    }
    // group g is the run [start[g], start[g + 1])
    for (int g = threadIdx.x; g <= a.n_groups; g += blockDim.x)
        start[g] = lower_bound_u64(keys, a.n, (uint64_t)g << kNormGroupShift);
    __syncthreads();
    constexpr uint64_t kIdxMask = (1ull << kNormIdxBits) - 1ull;
    if (a.mode == 0) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, waves = blockDim.x >> 6;
        for (int g = wave; g < a.n_groups; g += waves) {
            const int s0 = start[g], s1 = start[g + 1], c = s1 - s0;
            if (c == 0) continue;
            double part = 0.0;
            for (int p = s0 + lane; p < s1; p += 64)
                part += (double)from_order_bits((uint32_t)(keys[p] >> kNormValShift));
            const double mu = wave_sum(part) / (double)c;
            part = 0.0;
            for (int p = s0 + lane; p < s1; p += 64) {
                const double dev = (double)from_order_bits((uint32_t)(keys[p] >> kNormValShift)) - mu;
                part += dev * dev;
            }
            const double sd = __builtin_sqrt(wave_sum(part) / (double)c);
            for (int p = s0 + lane; p < s1; p += 64) {
                const int i = (int)(keys[p] & kIdxMask);
                a.out[i] = sd > 0.0 ? (float)(((double)a.r[i] - mu) / sd) : 0.0f;
            }
        }
    } else {
        for (int p = threadIdx.x; p < a.n; p += blockDim.x) {
            const uint64_t key = keys[p];
            const int g = (int)(key >> kNormGroupShift);
            const uint64_t first = key & ~kIdxMask;           // (group, value, index 0)
            const int lo = lower_bound_u64(keys, a.n, first);
            const int hi = lower_bound_u64(keys, a.n, first + (kIdxMask + 1));
            const int c = start[g + 1] - start[g];
            float o = 0.0f;
            if (c > 1) {
                const double rank = (double)(lo - start[g]) + 0.5 * (double)(hi - lo - 1);
                o = (float)(rank / (double)(c - 1) - 0.5);
            }
            a.out[(int)(key & kIdxMask)] = o;
        }
    }
    if (a.status && threadIdx.x == 0) *a.status = 0;
}

// -------------------------------------------------------------- partition --
// Keyed Feistel permutation of [0, 2^(2h)), eight rounds, round function =
// word 0 of Philox block (counter (R, r, 3, 0), key seed); cycle-walked into
// [0, d).
constexpr int kFeistelRounds = 8;
constexpr int kMaxWalk = 1 << 16;

__device__ __forceinline__ uint64_t feistel(uint32_t k0, uint32_t k1, int h, uint64_t x)
{
    const uint64_t mask = (1ull << h) - 1ull;
    uint64_t L = x >> h, R = x & mask;
#pragma unroll
    for (int r = 0; r < kFeistelRounds; ++r) {
        const Words4 y = philox4x32_10((uint32_t)R, (uint32_t)r, 3u, 0u, k0, k1);
        const uint64_t nr = L ^ ((uint64_t)y.x & mask);
        L = R;
        R = nr;
    }
    return (L << h) | R;
}

__device__ __forceinline__ uint64_t prp(uint32_t k0, uint32_t k1, int h, uint64_t d, uint64_t x, bool& overflow)
{
    uint64_t y = feistel(k0, k1, h, x);
    int walk = 0;
    while (y >= d) {
        y = feistel(k0, k1, h, y);
        if (++walk >= kMaxWalk) {
            overflow = true;
            y = 0;
            break;
        }
    }
    return y;
}

__global__ void k_status_zero(int32_t* status)
{
    if (status) *status = 0;
}

// Pass 1: bucket of every element, and per-tile bucket counts.
__global__ __launch_bounds__(kBlock) void k_part_bucket(PartitionArgs a)
{
    __shared__ uint32_t hist[kBlock / 64][256];
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    for (int k = lane; k < 256; k += 64) hist[wave][k] = 0;
    __builtin_amdgcn_wave_barrier();
    const int64_t tile = (int64_t)blockIdx.x * (kBlock / 64) + wave;
    if (tile >= a.n_tiles) return;
    bool overflow = false;
    for (int it = 0; it < kTileItems; ++it) {
        const int64_t e = tile * kTile + (int64_t)it * 64 + lane;
        if (e < a.d) {
            const uint64_t y = prp(k0, k1, a.half_bits, (uint64_t)a.d, (uint64_t)e, overflow);
            const uint32_t b = (uint32_t)((y * (uint64_t)a.K) / (uint64_t)a.d);
            a.bucket[e] = (uint8_t)b;
            atomicAdd(&hist[wave][b], 1u);
        }
    }
    if (overflow && a.status) atomicOr(a.status, 1);
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    for (int k = lane; k < a.K; k += 64) a.counts[(int64_t)k * a.n_tiles + tile] = hist[wave][k];
}

// Scan pass A: sum of each chunk of kScanChunk counts.
__global__ __launch_bounds__(kBlock) void k_scan_reduce(const uint32_t* counts, int64_t n, int64_t* block_sums)
{
    __shared__ int64_t part[kBlock];
    const int64_t base = (int64_t)blockIdx.x * kScanChunk;
    int64_t s = 0;
    for (int k = threadIdx.x; k < kScanChunk; k += kBlock)
        if (base + k < n) s += counts[base + k];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int off = kBlock / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) part[threadIdx.x] += part[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) block_sums[blockIdx.x] = part[0];
}

// Block-wide exclusive scan of kBlock values held one per thread.
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t v, int64_t* tmp, int64_t& total)
{
    tmp[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < kBlock; off <<= 1) {
        const int64_t add = threadIdx.x >= (unsigned)off ? tmp[threadIdx.x - off] : 0;
        __syncthreads();
        tmp[threadIdx.x] += add;
        __syncthreads();
    }
    total = tmp[kBlock - 1];
    const int64_t incl = tmp[threadIdx.x];
    __syncthreads();
    return incl - v;
}

// Scan pass B: exclusive scan of the chunk sums, in place (one workgroup).
__global__ __launch_bounds__(kBlock) void k_scan_blocks(int64_t* block_sums, int64_t nb)
{
    __shared__ int64_t tmp[kBlock];
    int64_t carry = 0;
    for (int64_t base = 0; base < nb; base += kBlock) {
        const int64_t i = base + threadIdx.x;
        const int64_t v = i < nb ? block_sums[i] : 0;
        int64_t total;
        const int64_t ex = block_exclusive_scan(v, tmp, total);
        if (i < nb) block_sums[i] = carry + ex;
        carry += total;
    }
}

// Scan pass C: exclusive positions of every count.
__global__ __launch_bounds__(kBlock) void k_scan_down(const uint32_t* counts, int64_t n, const int64_t* block_sums,
                                                      int64_t* pos)
{
    __shared__ int64_t tmp[kBlock];
    constexpr int per = kScanChunk / kBlock;   // consecutive entries per thread
    const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * per;
    int64_t v[per];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < per; ++k) {
        v[k] = base + k < n ? counts[base + k] : 0;
        s += v[k];
    }
    int64_t total;
    int64_t run = block_sums[blockIdx.x] + block_exclusive_scan(s, tmp, total);
#pragma unroll
    for (int k = 0; k < per; ++k) {
        if (base + k < n) pos[base + k] = run;
        run += v[k];
    }
}

// Pass 3: stable scatter.  Each wave walks its tile in element order, ranks
// the 64 elements of a step among equal buckets with ballots, and appends them
// to each bucket's run.
__global__ __launch_bounds__(kBlock) void k_part_scatter(PartitionArgs a)
{
    __shared__ int64_t base[kBlock / 64][256];
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int64_t tile = (int64_t)blockIdx.x * (kBlock / 64) + wave;
    if (tile >= a.n_tiles) return;
    for (int k = lane; k < a.K; k += 64) base[wave][k] = a.pos[(int64_t)k * a.n_tiles + tile];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    int nbits = 0;
    while ((1 << nbits) < a.K) ++nbits;
    const uint64_t below = (1ull << lane) - 1ull;
    for (int it = 0; it < kTileItems; ++it) {
        const int64_t e = tile * kTile + (int64_t)it * 64 + lane;
        const bool valid = e < a.d;
        const uint32_t b = valid ? a.bucket[e] : 0u;
        uint64_t same = __ballot(valid);
        for (int bit = 0; bit < nbits; ++bit) {
            const uint64_t m = __ballot((b >> bit) & 1u);
            same &= ((b >> bit) & 1u) ? m : ~m;
        }
        const int rank = __popcll(same & below);
        if (valid) {
            if (a.index32)
                a.index32[base[wave][b] + rank] = (uint32_t)e;
            else
                a.index[base[wave][b] + rank] = e;
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        if (valid && rank == 0) base[wave][b] += __popcll(same);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
}

// ------------------------------------------------------------------ debug --
__global__ __launch_bounds__(kBlock) void k_debug_philox(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks,
                                                         uint32_t* out)
{
    for (int64_t b = global_tid(); b < nblocks; b += grid_stride()) {
        const Words4 x = stream_block((uint32_t)seed, (uint32_t)(seed >> 32), domain, q0 + (uint64_t)b);
        reinterpret_cast<uint4*>(out)[b] = make_uint4(x.x, x.y, x.z, x.w);
    }
}

__global__ __launch_bounds__(kBlock) void k_debug_normals(uint64_t seed, int64_t j0, int64_t n, float* out)
{
    const BmTables* tb = stage_bm_tables<kBlock>();
    const int64_t qa = j0 >> 2;                      // first block touched
    const int64_t qb = (j0 + n + 3) >> 2;            // one past the last
    for (int64_t q = qa + global_tid(); q < qb; q += grid_stride()) {
        float z[4];
        normals4((uint32_t)seed, (uint32_t)(seed >> 32), (uint64_t)q, tb, z);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int64_t j = 4 * q + t;
            if (j >= j0 && j < j0 + n) out[j - j0] = z[t];
        }
    }
}

// Seeded normal fill: w[j] = cast(stddev * z_j), z_j the normal of position
// j in stream (seed, domain).
template <typename T, bool VEC>
__global__ __launch_bounds__(kBlock) void k_fill_normal(T* w, int64_t n, uint64_t seed, uint32_t domain, float stddev)
{
    constexpr int N = UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    auto body = [&](int64_t u, bool vec) {
        const int64_t j0 = u * N;
        float z[N];
        if (N == 8)
            normals8(k0, k1, (uint64_t)j0 >> 2, tb, z, domain);
        else
            normals4(k0, k1, (uint64_t)j0 >> 2, tb, z, domain);
        T v[N];
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = from_f32<T>(stddev * z[e]);
        if (vec) {
            store_vec<T>(w + j0, v);
        } else {
#pragma unroll
            for (int e = 0; e < N; ++e)
                if (j0 + e < n) w[j0 + e] = v[e];
        }
    };
    const int64_t full = n / N;
    for (int64_t u = global_tid(); u < full; u += grid_stride()) body(u, VEC);
    if (full * N < n && global_tid() == 0) body(full, false);
}

__global__ __launch_bounds__(kBlock) void k_debug_bm_grid(uint32_t m0, int64_t n, double* rho, double* c, double* s)
{
    const BmTables* tb = stage_bm_tables<kBlock>();
    for (int64_t k = global_tid(); k < n; k += grid_stride()) {
        const uint32_t word = (m0 + (uint32_t)k - 1u) << 8;
        if (rho) rho[k] = bm_radius(word, tb);
        double cc, ss;
        bm_angle(word, tb, cc, ss);
        if (c) c[k] = cc;
        if (s) s[k] = ss;
    }
}

__global__ __launch_bounds__(kBlock) void k_debug_prp(uint64_t seed, int64_t d, int32_t K, int32_t h, int64_t i0,
                                                      int64_t n, int64_t* perm, int32_t* bucket)
{
    for (int64_t k = global_tid(); k < n; k += grid_stride()) {
        bool overflow = false;
        const uint64_t y = prp((uint32_t)seed, (uint32_t)(seed >> 32), h, (uint64_t)d, (uint64_t)(i0 + k), overflow);
        if (perm) perm[k] = (int64_t)y;
        if (bucket) bucket[k] = (int32_t)((y * (uint64_t)K) / (uint64_t)d);
    }
}

__global__ void k_zero_u32(uint32_t* p)
{
    *p = 0u;
}

// RNG-only probe: each thread takes units of 8 positions and, like the update,
// generates the noise of kRngProbeStreams consecutive seeds for each unit into
// 8 independent fp32 accumulators; the accumulators' bits are folded into one
// word at the end.  No memory traffic but one atomic per wave.
constexpr int kRngProbeStreams = 16;

__global__ __launch_bounds__(kBlock) void k_rng_probe(uint64_t seed, int64_t units, uint32_t* sink)
{
    const BmTables* tb = stage_bm_tables<kBlock>();
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
    for (int64_t u = global_tid(); u < units; u += grid_stride()) {
        for (int st = 0; st < kRngProbeStreams; ++st) {
            const uint64_t key = seed + (uint64_t)st;
            float z[8];
            normals8((uint32_t)key, (uint32_t)(key >> 32), (uint64_t)u * 2u, tb, z);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = __builtin_fmaf(0.5f, z[e], acc[e]);
        }
    }
    uint32_t x = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) x ^= __float_as_uint(acc[e]);
    for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off);
    if ((threadIdx.x & 63) == 0) atomicXor(sink, x);
}

// Measurement references with nothing but the memory traffic.  The plainest
// gather (DIR 0: buf[j] = w[p(j)]) or scatter (DIR 1: w[p(j)] = buf[j])
// through an element map, one position per thread.
template <typename T, int DIR, int ADDR>
__global__ __launch_bounds__(kBlock) void k_probe_map_copy(StreamArgs a)
{
    T* w = static_cast<T*>(a.w);
    T* buf = static_cast<T*>(a.aux);
    for (int64_t j = global_tid(); j < a.length; j += grid_stride()) {
        const int64_t i = map_entry<ADDR>(a.index, a.offset + j);
        if ((uint64_t)i >= (uint64_t)a.numel) continue;
        if (DIR == 0)
            buf[j] = w[i];
        else
            w[i] = buf[j];
    }
}

// A plain copy of n16 16-byte vectors, one per thread per iteration; NT
// takes non-temporal loads and stores.
template <bool NT>
__global__ __launch_bounds__(kBlock) void k_probe_copy(const V4u* src, V4u* dst, int64_t n16)
{
    for (int64_t i = global_tid(); i < n16; i += grid_stride()) {
        if (NT)
            __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
        else
            dst[i] = src[i];
    }
}

int64_t grid_for(int64_t work_items, int64_t cap = kMaxGrid)
{
    int64_t blocks = (work_items + kBlock - 1) / kBlock;
    if (blocks < 1) blocks = 1;
    return blocks < cap ? blocks : cap;
}

// Noise kernels on contiguous or chunked subspaces loop over the subspace from
// a few workgroups per CU (the tables are staged once per workgroup).
template <typename K, typename A>
hipError_t launch1d(K kernel, int64_t items, const A& args, hipStream_t s, int64_t cap)
{
    hipLaunchKernelGGL(kernel, dim3((unsigned)grid_for(items, cap)), dim3(kBlock), 0, s, args);
    return hipGetLastError();
}

template <typename T>
int64_t units_of(int64_t length)
{
    return (length + UnitOf<T>::n - 1) / UnitOf<T>::n;
}

// Map kernels: one wave per tile of 64 N positions, up to the grid cap; the
// waves of a launch then start in position order, which keeps the scattered
// accesses in flight within a narrow window of the weights.
template <typename T>
int64_t map_threads(int64_t length)
{
    const int64_t tile = 64 * UnitOf<T>::n;
    return (length + tile - 1) / tile * 64;
}

// Instantiate a streaming kernel for the addressing mode and vector flag;
// element maps go to the map kernel MAPK instantiated with MARGS.
#define CPES_DISPATCH(KERNEL, KARGS, MAPK, MARGS)                                                     \
    switch (addr) {                                                                                  \
    case kGather: return launch1d(MAPK<MARGS, kGather>, map_threads<T>(a.length), a, s, kMaxGrid); \
    case kGather32: return launch1d(MAPK<MARGS, kGather32>, map_threads<T>(a.length), a, s, kMaxGrid); \
    case kChunk: return vec ? launch1d(KERNEL<KARGS, kChunk, true>, u, a, s, cap)                    \
                            : launch1d(KERNEL<KARGS, kChunk, false>, u, a, s, cap);                  \
    default: return vec ? launch1d(KERNEL<KARGS, kContig, true>, u, a, s, cap)                       \
                        : launch1d(KERNEL<KARGS, kContig, false>, u, a, s, cap);                     \
    }
#define CPES_COMMA ,

// Dense-window kernels (ascending maps, bf16): one wave per tile of kDenseTile entries.
int64_t dense_threads(int64_t length)
{
    return (length + kDenseTile - 1) / kDenseTile * 64;
}

template <typename T, int AUX>
hipError_t perturb_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    if (std::is_same<T, uint16_t>::value && a.dense) {
        const dim3 grid((unsigned)std::min<int64_t>(std::max<int64_t>((dense_threads(a.length) + kDenseBlock - 1) / kDenseBlock, 1),
                                                    kRngMaxGrid / 2));
        if (addr == kGather) hipLaunchKernelGGL((k_perturb_dense<AUX, kGather>), grid, dim3(kDenseBlock), 0, s, a);
        else if (addr == kGather32) hipLaunchKernelGGL((k_perturb_dense<AUX, kGather32>), grid, dim3(kDenseBlock), 0, s, a);
        if (addr == kGather || addr == kGather32) return hipGetLastError();
    }
    const int64_t u = units_of<T>(a.length), cap = kRngMaxGrid;
    if (vec) {
        CPES_DISPATCH(k_perturb, T CPES_COMMA AUX, k_perturb_map, T CPES_COMMA AUX CPES_COMMA true)
    }
    CPES_DISPATCH(k_perturb, T CPES_COMMA AUX, k_perturb_map, T CPES_COMMA AUX CPES_COMMA false)
}

template <typename T, bool MASTER>
hipError_t update_t(int addr, bool vec, const UpdateArgs& a, hipStream_t s)
{
    constexpr int N = MASTER ? 8 : UnitOf<T>::n;
    const int64_t u = (a.length + N - 1) / N, cap = kRngMaxGrid;
    if (vec) {
        CPES_DISPATCH(k_update, T CPES_COMMA MASTER, k_update_map, T CPES_COMMA MASTER CPES_COMMA true)
    }
    CPES_DISPATCH(k_update, T CPES_COMMA MASTER, k_update_map, T CPES_COMMA MASTER CPES_COMMA false)
}

// Copies whose source and destination together exceed the 256 MB last-level
// cache take the non-temporal loads and stores.
constexpr int64_t kStreamingBytes = 256ll << 20;

inline bool streaming(int64_t length, int bytes_per_position)
{
    return length * bytes_per_position > kStreamingBytes;
}

template <typename T>
hipError_t restore_copy_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    if (std::is_same<T, uint16_t>::value && a.dense) {
        if (addr == kGather) return launch1d(k_restore_dense<kCopyRestore, kGather>, dense_threads(a.length), a, s, kMaxGrid);
        if (addr == kGather32) return launch1d(k_restore_dense<kCopyRestore, kGather32>, dense_threads(a.length), a, s, kMaxGrid);
    }
    const int64_t u = units_of<T>(a.length), cap = kMaxGrid;
    if (streaming(a.length, 2 * sizeof(T))) {
        CPES_DISPATCH(k_restore_copy, T CPES_COMMA true, k_copy_map, T CPES_COMMA kCopyRestore CPES_COMMA true)
    }
    CPES_DISPATCH(k_restore_copy, T CPES_COMMA false, k_copy_map, T CPES_COMMA kCopyRestore CPES_COMMA false)
}

template <typename T>
hipError_t backup_copy_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    const int64_t u = units_of<T>(a.length), cap = kMaxGrid;
    if (streaming(a.length, 2 * sizeof(T))) {
        CPES_DISPATCH(k_backup_copy, T CPES_COMMA true, k_copy_map, T CPES_COMMA kCopyBackup CPES_COMMA true)
    }
    CPES_DISPATCH(k_backup_copy, T CPES_COMMA false, k_copy_map, T CPES_COMMA kCopyBackup CPES_COMMA false)
}

template <typename T>
hipError_t stage_master_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    const int64_t u = units_of<T>(a.length), cap = kMaxGrid;
    if (streaming(a.length, sizeof(T) + 4)) {
        CPES_DISPATCH(k_stage_master, T CPES_COMMA true, k_copy_map, T CPES_COMMA kCopyStageMaster CPES_COMMA true)
    }
    CPES_DISPATCH(k_stage_master, T CPES_COMMA false, k_copy_map, T CPES_COMMA kCopyStageMaster CPES_COMMA false)
}

hipError_t restore_master_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    using T = uint16_t;
    if (a.dense) {
        if (addr == kGather) return launch1d(k_restore_dense<kCopyRestoreMaster, kGather>, dense_threads(a.length), a, s, kMaxGrid);
        if (addr == kGather32) return launch1d(k_restore_dense<kCopyRestoreMaster, kGather32>, dense_threads(a.length), a, s, kMaxGrid);
    }
    const int64_t u = (a.length + 7) / 8, cap = kMaxGrid;
    if (streaming(a.length, 6)) {
        CPES_DISPATCH(k_restore_master, true, k_copy_map, T CPES_COMMA kCopyRestoreMaster CPES_COMMA true)
    }
    CPES_DISPATCH(k_restore_master, false, k_copy_map, T CPES_COMMA kCopyRestoreMaster CPES_COMMA false)
}

template <typename T>
hipError_t update_step_t(int addr, const StepArgs& a, hipStream_t s)
{
    const bool map = addr == kGather || addr == kGather32;
    const int64_t blocks = grid_for(a.tile_begin[a.K] * 64, map ? kMaxGrid : kRngMaxGrid);
    switch (addr) {
    case kGather: hipLaunchKernelGGL((k_update_step<T, kGather>), dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
    case kGather32: hipLaunchKernelGGL((k_update_step<T, kGather32>), dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
    case kChunk: hipLaunchKernelGGL((k_update_step<T, kChunk>), dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
    default: hipLaunchKernelGGL((k_update_step<T, kContig>), dim3((unsigned)blocks), dim3(kBlock), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_perturb(int dtype, int aux, int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    if (dtype == 0) {
        if (aux == kAuxSnapshot) return perturb_t<uint16_t, kAuxSnapshot>(addr, vec, a, s);
        if (aux == kAuxMaster) return perturb_t<uint16_t, kAuxMaster>(addr, vec, a, s);
        if (aux == kAuxBackup) return perturb_t<uint16_t, kAuxBackup>(addr, vec, a, s);
        return perturb_t<uint16_t, kAuxNone>(addr, vec, a, s);
    }
    if (aux == kAuxSnapshot) return perturb_t<float, kAuxSnapshot>(addr, vec, a, s);
    if (aux == kAuxBackup) return perturb_t<float, kAuxBackup>(addr, vec, a, s);
    return perturb_t<float, kAuxNone>(addr, vec, a, s);
}

hipError_t launch_restore_copy(int dtype, int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    return dtype == 0 ? restore_copy_t<uint16_t>(addr, vec, a, s) : restore_copy_t<float>(addr, vec, a, s);
}

hipError_t launch_backup_copy(int dtype, int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    return dtype == 0 ? backup_copy_t<uint16_t>(addr, vec, a, s) : backup_copy_t<float>(addr, vec, a, s);
}

hipError_t launch_restore_master(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    return restore_master_t(addr, vec, a, s);
}

hipError_t launch_stage_master(int dtype, int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    return dtype == 0 ? stage_master_t<uint16_t>(addr, vec, a, s) : stage_master_t<float>(addr, vec, a, s);
}

hipError_t launch_update(int dtype, bool master, int addr, bool vec, const UpdateArgs& a, hipStream_t s)
{
    if (dtype == 0) return master ? update_t<uint16_t, true>(addr, vec, a, s) : update_t<uint16_t, false>(addr, vec, a, s);
    return update_t<float, false>(addr, vec, a, s);
}

hipError_t launch_update_step(int dtype, int addr, const StepArgs& a, hipStream_t s)
{
    return dtype == 0 ? update_step_t<uint16_t>(addr, a, s) : update_step_t<float>(addr, a, s);
}

hipError_t launch_fill_normal(int dtype, void* w, int64_t n, uint64_t seed, uint32_t domain, float stddev, bool vec,
                              hipStream_t s)
{
    const dim3 grid((unsigned)grid_for(n / (dtype == 0 ? 8 : 4) + 1, kRngMaxGrid)), block(kBlock);
    if (dtype == 0) {
        uint16_t* p = static_cast<uint16_t*>(w);
        if (vec) hipLaunchKernelGGL((k_fill_normal<uint16_t, true>), grid, block, 0, s, p, n, seed, domain, stddev);
        else hipLaunchKernelGGL((k_fill_normal<uint16_t, false>), grid, block, 0, s, p, n, seed, domain, stddev);
    } else {
        float* p = static_cast<float*>(w);
        if (vec) hipLaunchKernelGGL((k_fill_normal<float, true>), grid, block, 0, s, p, n, seed, domain, stddev);
        else hipLaunchKernelGGL((k_fill_normal<float, false>), grid, block, 0, s, p, n, seed, domain, stddev);
    }
    return hipGetLastError();
}

hipError_t launch_normalize(const NormalizeArgs& a, hipStream_t s)
{
    hipLaunchKernelGGL(k_normalize, dim3(1), dim3(kNormThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_partition(const PartitionArgs& a, hipStream_t s)
{
    const int64_t waves_per_block = kBlock / 64;
    const unsigned tile_blocks = (unsigned)((a.n_tiles + waves_per_block - 1) / waves_per_block);
    const int64_t n_counts = (int64_t)a.K * a.n_tiles;
    const unsigned scan_blocks = (unsigned)((n_counts + kScanChunk - 1) / kScanChunk);
    hipLaunchKernelGGL(k_status_zero, dim3(1), dim3(1), 0, s, a.status);
    hipLaunchKernelGGL(k_part_bucket, dim3(tile_blocks), dim3(kBlock), 0, s, a);
    hipLaunchKernelGGL(k_scan_reduce, dim3(scan_blocks), dim3(kBlock), 0, s, a.counts, n_counts, a.block_sums);
    hipLaunchKernelGGL(k_scan_blocks, dim3(1), dim3(kBlock), 0, s, a.block_sums, (int64_t)scan_blocks);
    hipLaunchKernelGGL(k_scan_down, dim3(scan_blocks), dim3(kBlock), 0, s, a.counts, n_counts, a.block_sums, a.pos);
    hipLaunchKernelGGL(k_part_scatter, dim3(tile_blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_debug_philox(uint64_t seed, uint32_t domain, uint64_t q0, int64_t nblocks, uint32_t* out, hipStream_t s)
{
    hipLaunchKernelGGL(k_debug_philox, dim3((unsigned)grid_for(nblocks)), dim3(kBlock), 0, s, seed, domain, q0, nblocks, out);
    return hipGetLastError();
}

hipError_t launch_debug_normals(uint64_t seed, int64_t j0, int64_t n, float* out, hipStream_t s)
{
    const int64_t blocks = ((j0 + n + 3) >> 2) - (j0 >> 2);
    hipLaunchKernelGGL(k_debug_normals, dim3((unsigned)grid_for(blocks, kRngMaxGrid)), dim3(kBlock), 0, s, seed, j0, n, out);
    return hipGetLastError();
}

hipError_t launch_debug_bm_grid(uint32_t m0, int64_t n, double* rho, double* c, double* sn, hipStream_t s)
{
    hipLaunchKernelGGL(k_debug_bm_grid, dim3((unsigned)grid_for(n, kRngMaxGrid)), dim3(kBlock), 0, s, m0, n, rho, c, sn);
    return hipGetLastError();
}

hipError_t launch_debug_prp(uint64_t seed, int64_t d, int32_t K, int32_t half_bits, int64_t i0, int64_t n,
                            int64_t* perm, int32_t* bucket, hipStream_t s)
{
    hipLaunchKernelGGL(k_debug_prp, dim3((unsigned)grid_for(n)), dim3(kBlock), 0, s, seed, d, K, half_bits, i0, n,
                       perm, bucket);
    return hipGetLastError();
}

hipError_t launch_rng_probe(uint64_t seed, int64_t n, uint32_t* sink, hipStream_t s)
{
    // a few workgroups per CU looping over the units: one atomic per wave
    const int64_t units = (n + 8 * kRngProbeStreams - 1) / (8 * kRngProbeStreams);
    const int64_t blocks = grid_for(units, kRngMaxGrid);
    hipLaunchKernelGGL(k_zero_u32, dim3(1), dim3(1), 0, s, sink);
    hipLaunchKernelGGL(k_rng_probe, dim3((unsigned)blocks), dim3(kBlock), 0, s, seed, units, sink);
    return hipGetLastError();
}

hipError_t launch_probe_map_copy(int dtype, int addr, int direction, const StreamArgs& a, hipStream_t s)
{
    const int64_t g = grid_for(a.length);
#define CPES_PROBE(T, D, A) hipLaunchKernelGGL((k_probe_map_copy<T, D, A>), dim3((unsigned)g), dim3(kBlock), 0, s, a)
    if (dtype == 0) {
        if (addr == kGather32) {
            if (direction == 0) CPES_PROBE(uint16_t, 0, kGather32); else CPES_PROBE(uint16_t, 1, kGather32);
        } else {
            if (direction == 0) CPES_PROBE(uint16_t, 0, kGather); else CPES_PROBE(uint16_t, 1, kGather);
        }
    } else {
        if (addr == kGather32) {
            if (direction == 0) CPES_PROBE(float, 0, kGather32); else CPES_PROBE(float, 1, kGather32);
        } else {
            if (direction == 0) CPES_PROBE(float, 0, kGather); else CPES_PROBE(float, 1, kGather);
        }
    }
#undef CPES_PROBE
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void* src, void* dst, int64_t bytes, bool nontemporal, hipStream_t s)
{
    const int64_t n16 = bytes / 16;
    const dim3 grid((unsigned)grid_for(n16)), block(kBlock);
    if (nontemporal)
        hipLaunchKernelGGL(k_probe_copy<true>, grid, block, 0, s, static_cast<const V4u*>(src), static_cast<V4u*>(dst), n16);
    else
        hipLaunchKernelGGL(k_probe_copy<false>, grid, block, 0, s, static_cast<const V4u*>(src), static_cast<V4u*>(dst), n16);
    return hipGetLastError();
}

}  // namespace cpes
