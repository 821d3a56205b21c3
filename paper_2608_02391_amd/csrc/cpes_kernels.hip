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
template <int N>
__device__ __forceinline__ void load_index(const int64_t* p, int64_t v[N])
{
#pragma unroll
    for (int h = 0; h < N / 2; ++h) {
        const longlong2 x = reinterpret_cast<const longlong2*>(p)[h];
        v[2 * h] = x.x;
        v[2 * h + 1] = x.y;
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

// The map entries of positions p .. p + N - 1 (16-byte loads; p + index must
// be 16-byte aligned), widened to int64.
template <int ADDR, int N>
__device__ __forceinline__ void load_map(const int64_t* index, int64_t p, int64_t v[N])
{
    if (ADDR == kGather) {
        load_index<N>(index + p, v);
    } else {
        const uint4* q = reinterpret_cast<const uint4*>(reinterpret_cast<const uint32_t*>(index) + p);
#pragma unroll
        for (int h = 0; h < N / 4; ++h) {
            const uint4 x = q[h];
            v[4 * h + 0] = x.x; v[4 * h + 1] = x.y; v[4 * h + 2] = x.z; v[4 * h + 3] = x.w;
        }
    }
}

// Scatter one unit through a map.  When every entry is valid (always, for a
// partition's own map) the stores run without per-element branches, so they
// issue back to back: with a branch around each store the wait for the loaded
// data is repeated before every store and, since stores share the vector
// memory counter, each store then waits for the one before it.
template <typename T, int N>
__device__ __forceinline__ void scatter_unit(T* w, const int64_t idx[N], const T v[N], int64_t numel)
{
    uint32_t bad = 0;   // bitwise, not short-circuit: keeps the check free of branches
#pragma unroll
    for (int e = 0; e < N; ++e) bad |= (uint64_t)idx[e] >= (uint64_t)numel ? 1u : 0u;
    if (bad == 0) {
#pragma unroll
        for (int e = 0; e < N; ++e) w[idx[e]] = v[e];
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e)
            if (idx[e] >= 0 && idx[e] < numel) w[idx[e]] = v[e];
    }
}

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
// replay restore with scale = -sign * sigma.
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
        int64_t idx[N];
        if (kMap<ADDR>) {
            load_map<ADDR, N>(a.index, a.offset + j0, idx);
        } else if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
            scalar_body(u);
            return;
        }
        float src[N];
        T old[N];
        if (kMap<ADDR> && AUX != kAuxMaster && AUX != kAuxBackup) {
#pragma unroll
            for (int e = 0; e < N; ++e) {
                const bool ok = idx[e] >= 0 && idx[e] < a.numel;
                old[e] = ok ? w[idx[e]] : T(0);
            }
        } else if (AUX != kAuxMaster && AUX != kAuxBackup) {
            load_vec<T>(w + base, old);
        }
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
        if (kMap<ADDR>) {
            scatter_unit<T, N>(w, idx, out, a.numel);
        } else {
            store_vec<T>(w + base, out);
        }
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
        T v[N];
        load_vec<T, NT>(snap + j0, v);
        if (kMap<ADDR>) {
            int64_t idx[N];
            load_map<ADDR, N>(a.index, a.offset + j0, idx);
            scatter_unit<T, N>(w, idx, v, a.numel);
        } else {
            int64_t base;
            if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
                scalar_body(u);
                return;
            }
            store_vec<T, NT>(w + base, v);
        }
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
        T v[N];
        if (kMap<ADDR>) {
            int64_t idx[N];
            load_map<ADDR, N>(a.index, a.offset + j0, idx);
#pragma unroll
            for (int e = 0; e < N; ++e) v[e] = (idx[e] >= 0 && idx[e] < a.numel) ? w[idx[e]] : T(0);
        } else {
            int64_t base;
            if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
                scalar_body(u);
                return;
            }
            load_vec<T, NT>(w + base, v);
        }
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
        float m[N];
        load_f32s<N, NT>(master + j0, m);
        uint16_t v[N];
#pragma unroll
        for (int e = 0; e < N; ++e) v[e] = f32_to_bf16(m[e]);
        if (kMap<ADDR>) {
            int64_t idx[N];
            load_map<ADDR, N>(a.index, a.offset + j0, idx);
            scatter_unit<uint16_t, N>(w, idx, v, a.numel);
        } else {
            int64_t base;
            if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
                scalar_body(u);
                return;
            }
            store_vec<uint16_t, NT>(w + base, v);
        }
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
        T v[N];
        if (kMap<ADDR>) {
            int64_t idx[N];
            load_map<ADDR, N>(a.index, a.offset + j0, idx);
#pragma unroll
            for (int e = 0; e < N; ++e) v[e] = (idx[e] >= 0 && idx[e] < a.numel) ? w[idx[e]] : T(0);
        } else {
            int64_t base;
            if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
                scalar_body(u);
                return;
            }
            load_vec<T, NT>(w + base, v);
        }
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
template <typename T, bool MASTER, int ADDR, bool VEC>
__global__ __launch_bounds__(kBlock) void k_update(UpdateArgs a)
{
    constexpr int N = MASTER ? 8 : UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    __shared__ float coef[kMaxMembers];
    // Fold members into stream coefficients, in member order, in fp64.
    for (int u = threadIdx.x; u < a.n_streams; u += blockDim.x) {
        double c = 0.0;
        for (int i = 0; i < a.n_members; ++i)
            if (a.member_stream[i] == u) c += (double)a.member_sign[i] * (double)a.rnorm[i];
        coef[u] = (float)c;
    }
    __syncthreads();

    T* w = static_cast<T*>(a.w);
    auto accumulate = [&](int64_t j0, float acc[N]) {
#pragma unroll
        for (int e = 0; e < N; ++e) acc[e] = 0.0f;
        for (int s = 0; s < a.n_streams; ++s) {
            const float c = coef[s];
            float z[N];
            unit_normals<N>(a.seed_lo[s], a.seed_hi[s], (uint64_t)(a.noise0 + j0) >> 2, tb, z);
#pragma unroll
            for (int e = 0; e < N; ++e) acc[e] = __builtin_fmaf(c, z[e], acc[e]);
        }
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
        int64_t idx[N];
        int64_t base = 0;
        T v[N];
        if (kMap<ADDR>) {
            load_map<ADDR, N>(a.index, a.offset + j0, idx);
#pragma unroll
            for (int e = 0; e < N; ++e) v[e] = (idx[e] >= 0 && idx[e] < a.numel) ? w[idx[e]] : T(0);
        } else {
            if (!unit_base<ADDR>(a.index, a.offset, a.numel, a.chunk_shift, j0, N, base)) {
                scalar_finish(j0, acc);
                return;
            }
            if (!MASTER) load_vec<T>(w + base, v);
        }
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
        if (kMap<ADDR>) {
            scatter_unit<T, N>(w, idx, out, a.numel);
        } else {
            store_vec<T>(w + base, out);
        }
    };
    for_each_unit<N, VEC>(a.length, vec_body, scalar_body);
}

// ------------------------------------------------------------ step update --
// theta += sum_k P_k step_k sum_{u in streams of k} c_u eps_u (Eq. 13, Alg. 1):
// every subspace of the partition with its own members, in one launch.  Units
// restart at each subspace's first position, so noise position j is always
// relative to the subspace; each wave works on 64 units of one subspace.
template <typename T, int ADDR>
__global__ __launch_bounds__(kBlock) void k_update_step(StepArgs a)
{
    constexpr int N = UnitOf<T>::n;
    const BmTables* tb = stage_bm_tables<kBlock>();
    __shared__ float coef[kMaxMembers];
    for (int u = threadIdx.x; u < a.n_streams; u += blockDim.x) {
        double c = 0.0;
        for (int i = 0; i < a.n_members; ++i)
            if (a.member_stream[i] == u) c += (double)a.member_sign[i] * (double)a.rnorm[i];
        coef[u] = (float)c;
    }
    __syncthreads();
    T* w = static_cast<T*>(a.w);
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / 64);
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
    const int64_t tiles = a.tile_begin[a.K];
    for (int64_t t = wave; t < tiles; t += waves) {
        // t is the same for the whole wave; so are k and the stream range, which
        // keeps the seed and coefficient reads scalar
        int k = 0;
        while (k + 1 < a.K && a.tile_begin[k + 1] <= t) ++k;
        k = __builtin_amdgcn_readfirstlane(k);
        const int st0 = __builtin_amdgcn_readfirstlane(a.stream_begin[k]);
        const int st1 = __builtin_amdgcn_readfirstlane(a.stream_begin[k + 1]);
        const int64_t off = a.offset[k];
        const int64_t len = a.length[k];
        const int64_t j0 = ((t - a.tile_begin[k]) * 64 + lane) * N;
        if (j0 >= len) continue;
        int64_t base = 0;
        const bool vec = ((a.vec_mask >> k) & 1u) && j0 + N <= len &&
                         (kMap<ADDR> || unit_base<ADDR>(a.index, off, a.numel, a.chunk_shift, j0, N, base));
        float acc[N];
#pragma unroll
        for (int e = 0; e < N; ++e) acc[e] = 0.0f;
        for (int st = st0; st < st1; ++st) {
            const float c = coef[st];
            float z[N];
            unit_normals<N>(a.seed_lo[st], a.seed_hi[st], (uint64_t)j0 >> 2, tb, z);
#pragma unroll
            for (int e = 0; e < N; ++e) acc[e] = __builtin_fmaf(c, z[e], acc[e]);
        }
        const float step = a.step[k];
        if (vec) {
            T v[N], out[N];
            int64_t idx[N];
            if (kMap<ADDR>) {
                load_map<ADDR, N>(a.index, off + j0, idx);
#pragma unroll
                for (int e = 0; e < N; ++e) v[e] = (idx[e] >= 0 && idx[e] < a.numel) ? w[idx[e]] : T(0);
            } else {
                load_vec<T>(w + base, v);
            }
#pragma unroll
            for (int e = 0; e < N; ++e) out[e] = from_f32<T>(__builtin_fmaf(step, acc[e], to_f32<T>(v[e])));
            if (kMap<ADDR>) {
                scatter_unit<T, N>(w, idx, out, a.numel);
            } else {
                store_vec<T>(w + base, out);
            }
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
// One workgroup.  Group statistics are summed in fp64 in index order (one
// thread per group), exactly as the definition reads; ranks count smaller and
// equal rewards of the same group.
constexpr int kNormThreads = 256;
constexpr int kNormMaxN = 4096;
constexpr int kNormMaxGroups = 1024;

__global__ __launch_bounds__(kNormThreads) void k_normalize(NormalizeArgs a)
{
#pragma clang fp contract(off)
    __shared__ float r[kNormMaxN];
    __shared__ int32_t g[kNormMaxN];
    __shared__ double mu[kNormMaxGroups];
    __shared__ double sd[kNormMaxGroups];
    __shared__ int32_t cnt[kNormMaxGroups];
    __shared__ int bad;
    if (threadIdx.x == 0) bad = 0;
    __syncthreads();
    int my_bad = 0;
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        const float v = a.r[i];
        const int32_t gi = a.group ? a.group[i] : 0;
        r[i] = v;
        g[i] = gi;
        if (!__builtin_isfinite(v)) my_bad |= 1;
        if (gi < 0 || gi >= a.n_groups) my_bad |= 2;
    }
    if (my_bad) atomicOr(&bad, my_bad);
    __syncthreads();
    const int status = (bad & 2) ? 2 : (bad & 1) ? 1 : 0;
    if (status != 0) {
        for (int i = threadIdx.x; i < a.n; i += blockDim.x) a.out[i] = 0.0f;
        if (a.status && threadIdx.x == 0) *a.status = status;
        return;
    }
    for (int k = threadIdx.x; k < a.n_groups; k += blockDim.x) {
        int c = 0;
        double sum = 0.0;
        for (int j = 0; j < a.n; ++j)
            if (g[j] == k) {
                sum += (double)r[j];
                ++c;
            }
        cnt[k] = c;
        if (a.mode == 0 && c > 0) {
            const double m = sum / (double)c;
            double ss = 0.0;
            for (int j = 0; j < a.n; ++j)
                if (g[j] == k) {
                    const double dev = (double)r[j] - m;
                    const double sq = dev * dev;
                    ss += sq;
                }
            mu[k] = m;
            sd[k] = __builtin_sqrt(ss / (double)c);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < a.n; i += blockDim.x) {
        const int k = g[i];
        float o;
        if (a.mode == 0) {
            o = sd[k] > 0.0 ? (float)(((double)r[i] - mu[k]) / sd[k]) : 0.0f;
        } else {
            int less = 0, equal = 0;
            for (int j = 0; j < a.n; ++j) {
                if (g[j] != k) continue;
                less += r[j] < r[i];
                equal += r[j] == r[i];
            }
            const int c = cnt[k];
            if (c == 1) {
                o = 0.0f;
            } else {
                const double rank = (double)less + 0.5 * (double)(equal - 1);
                o = (float)(rank / (double)(c - 1) - 0.5);
            }
        }
        a.out[i] = o;
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

__global__ __launch_bounds__(kBlock) void k_rng_probe(uint64_t seed, int64_t n, uint32_t* sink)
{
    const BmTables* tb = stage_bm_tables<kBlock>();
    const int64_t units = (n + 7) / 8;
    uint32_t acc = 0;
    for (int64_t u = global_tid(); u < units; u += grid_stride()) {
        float z[8];
        normals8((uint32_t)seed, (uint32_t)(seed >> 32), (uint64_t)u * 2u, tb, z);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc ^= __float_as_uint(z[e]);
    }
    for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
    if ((threadIdx.x & 63) == 0) atomicXor(sink, acc);
}

int64_t grid_for(int64_t work_items, int64_t cap = kMaxGrid)
{
    int64_t blocks = (work_items + kBlock - 1) / kBlock;
    if (blocks < 1) blocks = 1;
    return blocks < cap ? blocks : cap;
}

// Noise kernels on contiguous or chunked subspaces loop over the subspace from
// a few workgroups per CU (the tables are staged once per workgroup).  On
// index maps one workgroup per 256 units is faster: workgroups then start in
// position order, so the scattered accesses in flight stay in a narrow window
// of the weights (DRAM row and cache locality).
inline int64_t rng_grid_cap(int addr)
{
    return addr == kGather || addr == kGather32 ? kMaxGrid : kRngMaxGrid;
}

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

// Instantiate a streaming kernel for the addressing mode and vector flag.
#define CPES_DISPATCH_ADDR_VEC(KERNEL, ...)                                                          \
    switch (addr) {                                                                                  \
    case kGather: return vec ? launch1d(KERNEL<__VA_ARGS__, kGather, true>, u, a, s, cap)                  \
                             : launch1d(KERNEL<__VA_ARGS__, kGather, false>, u, a, s, cap);                \
    case kGather32: return vec ? launch1d(KERNEL<__VA_ARGS__, kGather32, true>, u, a, s, cap)              \
                               : launch1d(KERNEL<__VA_ARGS__, kGather32, false>, u, a, s, cap);            \
    case kChunk: return vec ? launch1d(KERNEL<__VA_ARGS__, kChunk, true>, u, a, s, cap)                    \
                            : launch1d(KERNEL<__VA_ARGS__, kChunk, false>, u, a, s, cap);                  \
    default: return vec ? launch1d(KERNEL<__VA_ARGS__, kContig, true>, u, a, s, cap)                       \
                        : launch1d(KERNEL<__VA_ARGS__, kContig, false>, u, a, s, cap);                     \
    }

template <typename T, int AUX>
hipError_t perturb_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    const int64_t u = units_of<T>(a.length), cap = rng_grid_cap(addr);
    CPES_DISPATCH_ADDR_VEC(k_perturb, T, AUX)
}

template <typename T, bool MASTER>
hipError_t update_t(int addr, bool vec, const UpdateArgs& a, hipStream_t s)
{
    const int64_t u = (a.length + (MASTER ? 8 : UnitOf<T>::n) - 1) / (MASTER ? 8 : UnitOf<T>::n),
                  cap = rng_grid_cap(addr);
    CPES_DISPATCH_ADDR_VEC(k_update, T, MASTER)
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
    const int64_t u = units_of<T>(a.length), cap = kMaxGrid;
    if (streaming(a.length, 2 * sizeof(T))) {
        CPES_DISPATCH_ADDR_VEC(k_restore_copy, T, true)
    }
    CPES_DISPATCH_ADDR_VEC(k_restore_copy, T, false)
}

template <typename T>
hipError_t backup_copy_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    const int64_t u = units_of<T>(a.length), cap = kMaxGrid;
    if (streaming(a.length, 2 * sizeof(T))) {
        CPES_DISPATCH_ADDR_VEC(k_backup_copy, T, true)
    }
    CPES_DISPATCH_ADDR_VEC(k_backup_copy, T, false)
}

template <typename T>
hipError_t stage_master_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    const int64_t u = units_of<T>(a.length), cap = kMaxGrid;
    if (streaming(a.length, sizeof(T) + 4)) {
        CPES_DISPATCH_ADDR_VEC(k_stage_master, T, true)
    }
    CPES_DISPATCH_ADDR_VEC(k_stage_master, T, false)
}

hipError_t restore_master_t(int addr, bool vec, const StreamArgs& a, hipStream_t s)
{
    const int64_t u = (a.length + 7) / 8, cap = kMaxGrid;
    if (streaming(a.length, 6)) {
        CPES_DISPATCH_ADDR_VEC(k_restore_master, true)
    }
    CPES_DISPATCH_ADDR_VEC(k_restore_master, false)
}

template <typename T>
hipError_t update_step_t(int addr, const StepArgs& a, hipStream_t s)
{
    const int64_t blocks = grid_for(a.tile_begin[a.K] * 64, rng_grid_cap(addr));
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
    // A few workgroups per CU looping over the units: one atomic per wave.
    const int64_t blocks = grid_for((n + 7) / 8) < 8192 ? grid_for((n + 7) / 8) : 8192;
    hipLaunchKernelGGL(k_zero_u32, dim3(1), dim3(1), 0, s, sink);
    hipLaunchKernelGGL(k_rng_probe, dim3((unsigned)blocks), dim3(kBlock), 0, s, seed, n, sink);
    return hipGetLastError();
}

}  // namespace cpes
