// Device helpers shared by the wfstdec kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace wfd {

// Ordered key of a float32: unsigned order of keys equals numeric order,
// with -0 just below +0.  Costs are compared only through these keys.
__device__ __forceinline__ uint32_t okey(float x)
{
    uint32_t u = __float_as_uint(x);
    return (u >> 31) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float okey_val(uint32_t k)
{
    uint32_t u = (k >> 31) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// Token = cost key (high word) | user arc + 1 (low word); 0 marks the start
// token.  The unsigned minimum is the cheapest token, lowest arc on ties.
__device__ __forceinline__ uint64_t make_tok(uint32_t key, int32_t arc)
{
    return (static_cast<uint64_t>(key) << 32) | static_cast<uint32_t>(arc + 1);
}

__device__ __forceinline__ float tok_cost(uint64_t t) { return okey_val(static_cast<uint32_t>(t >> 32)); }
__device__ __forceinline__ int32_t tok_arc(uint64_t t) { return static_cast<int32_t>(static_cast<uint32_t>(t)) - 1; }

// Key of the largest cost a token may keep: fl(best + beam), never +inf.
__device__ __forceinline__ uint32_t beam_limit(uint32_t best_key, float beam)
{
    const uint32_t kmax = 0xFF7FFFFFu;   // okey(FLT_MAX)
    if (best_key == kEmptyKey) return kmax;
    uint32_t k = okey(okey_val(best_key) + beam);
    return k < kmax ? k : kmax;
}

// Early-drop bound during expansion: any candidate above fl(m + beam),
// m = a candidate cost already seen, can neither survive pruning nor lower a
// token that survives.
__device__ __forceinline__ uint32_t drop_bound(uint32_t m_key, float beam)
{
    if (m_key == kEmptyKey) return kEmptyKey;
    return okey(okey_val(m_key) + beam);
}

// Load through a pointer known to address device memory (a global rather
// than a flat access, which would also wait on LDS traffic).
template <typename T>
__device__ __forceinline__ T ldg(const T *ptr)
{
    return *(const __attribute__((address_space(1))) T *)ptr;
}

// Multiplicative hash of a state id for the open-addressing tables (the
// high bits index the table).
__device__ __forceinline__ uint32_t hash_state(uint32_t d, uint32_t mul) { return d * mul; }

// Order LDS stores of some lanes of a wave before loads of the same
// locations by other lanes of the wave: to the compiler such a hand-over is
// a data race unless fenced, and it may serve a lane's load from that lane's
// own earlier store.
__device__ __forceinline__ void wave_lds_handover()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int lane_id() { return static_cast<int>(__lane_id()); }

__device__ __forceinline__ uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

__device__ __forceinline__ int rank_in(uint64_t mask) { return __popcll(mask & lanemask_lt()); }

// Wave-wide inclusive sum with DPP lane moves (no LDS traffic): a
// Kogge-Stone scan inside each row of 16 lanes, then row 0's total into row
// 1 (and row 2's into row 3) and lane 31's into rows 2-3.  Lanes whose
// source lies outside the row read the identity.  Called by the whole wave.
__device__ __forceinline__ int wave_incl_scan(int x)
{
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);   // row_bcast:15
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return x;
}

// Wave-wide minimum (unsigned), the same lane moves; the result is lane 63's.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x)
{
    const int id = -1;   // identity: 0xFFFFFFFF
    x = min(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(id, static_cast<int>(x), 0x111, 0xf, 0xf, false)));
    x = min(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(id, static_cast<int>(x), 0x112, 0xf, 0xf, false)));
    x = min(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(id, static_cast<int>(x), 0x114, 0xf, 0xf, false)));
    x = min(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(id, static_cast<int>(x), 0x118, 0xf, 0xf, false)));
    x = min(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(id, static_cast<int>(x), 0x142, 0xa, 0xf, false)));
    x = min(x, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(id, static_cast<int>(x), 0x143, 0xc, 0xf, false)));
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x), kWave - 1));
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x)
{
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        uint64_t y = __shfl_xor(x, d, kWave);
        x = y < x ? y : x;
    }
    return x;
}

__device__ __forceinline__ long long wave_sum_ll(long long x)
{
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) x += __shfl_xor(x, d, kWave);
    return x;
}

// Largest lane l with pre[l] <= k, where pre is the exclusive prefix of
// per-lane counts (non-decreasing over lanes).  Called by the whole wave.
__device__ __forceinline__ int owner_lane(int pre, int k)
{
    int lo = 0, hi = kWave - 1;
#pragma unroll
    for (int it = 0; it < 6; it++) {
        int mid = (lo + hi + 1) >> 1;
        int pm = __shfl(pre, mid, kWave);
        if (pm <= k) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Owner lane of position k0 + lane (the same as owner_lane(pre, k0 + lane))
// for counts cnt whose exclusive prefix pre is non-decreasing over lanes,
// pre <= k0 in lane 0.  A lane whose first item lies at position 1..63 of the
// window sends its id there (ds_permute; a position no lane writes reads 0),
// position 0 takes the last lane whose first item is at most k0 (a ballot),
// and an inclusive maximum scan carries each owner over its items.  One LDS
// lane swizzle and six DPP steps instead of six dependent shuffles.  Called
// by the whole wave.
__device__ __forceinline__ int owner_scan(int pre, int cnt, int k0)
{
    const int lane = lane_id();
    const int s = pre - k0;
    const bool push = cnt > 0 && s > 0 && s < kWave;
    const int got = __builtin_amdgcn_ds_permute(push ? s * 4 : 0, push ? lane + 1 : 0);
    const uint64_t m = __ballot(pre <= k0);
    int v = lane == 0 ? kWave - __clzll(static_cast<long long>(m)) : got;
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false));   // row_shr:1
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false));   // row_shr:2
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false));   // row_shr:4
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false));   // row_shr:8
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false));   // row_bcast:15
    v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false));   // row_bcast:31
    return v - 1;
}

template <typename T>
__device__ __forceinline__ T ld_relaxed(T *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Barrier that orders LDS only: device-memory stores issued before it need
// not be complete.  Used where no other wave reads those stores before a
// full barrier.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wait until this wave's device-memory loads and stores have completed
// (s_waitcnt vmcnt(0); the other counters left free).  Before a barrier it
// makes the wave's stores visible in L2 to the block's later atomics and
// L2 loads, without the cache write-back and invalidation of a device-scope
// fence.
__device__ __forceinline__ void vm_wait() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Barrier after which the block's device-memory stores are complete.
__device__ __forceinline__ void block_sync_vm()
{
    vm_wait();
    __syncthreads();
}

__device__ __forceinline__ void set_status(UttState &st, int code)
{
    atomicCAS(&st.status, 0, code);
}

// Largest t in [0, n) with epre[t] <= a (epre non-decreasing, epre[0] <= a).
__device__ __forceinline__ int search_le(const int32_t *epre, int n, int a)
{
    const int lane = lane_id();
    int lo = 0, end = n;
    while (end - lo > 1) {
        const int step = (end - lo + kWave - 1) / kWave;
        const int idx = lo + lane * step;
        const int v = idx < end ? epre[idx] : 0x7FFFFFFF;
        const uint64_t m = __ballot(v <= a);
        const int l = 63 - __clzll(static_cast<long long>(m));
        lo += l * step;
        end = min(lo + step, end);
    }
    return lo;
}


// Three block-wide exclusive scans at once (blockDim.x a multiple of 64, at
// most 1024); `sh` needs 51 ints.  Returns the exclusive prefixes and stores
// the block totals in *total.
__device__ __forceinline__ int3 block_scan3(int x, int y, int z, int *sh, int3 *total)
{
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    const int ix = wave_incl_scan(x), iy = wave_incl_scan(y), iz = wave_incl_scan(z);
    if (lane == kWave - 1) {
        sh[w] = ix;
        sh[16 + w] = iy;
        sh[32 + w] = iz;
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
        const int vx = threadIdx.x < nw ? sh[threadIdx.x] : 0;
        const int vy = threadIdx.x < nw ? sh[16 + threadIdx.x] : 0;
        const int vz = threadIdx.x < nw ? sh[32 + threadIdx.x] : 0;
        const int sx = wave_incl_scan(vx), sy = wave_incl_scan(vy), sz = wave_incl_scan(vz);
        if (threadIdx.x < nw) {
            sh[threadIdx.x] = sx - vx;
            sh[16 + threadIdx.x] = sy - vy;
            sh[32 + threadIdx.x] = sz - vz;
        }
        if (threadIdx.x == kWave - 1) {
            sh[48] = sx;
            sh[49] = sy;
            sh[50] = sz;
        }
    }
    __syncthreads();
    const int3 r = make_int3(ix - x + sh[w], iy - y + sh[16 + w], iz - z + sh[32 + w]);
    *total = make_int3(sh[48], sh[49], sh[50]);
    __syncthreads();
    return r;
}

// Block-wide exclusive scan of one int per thread (blockDim.x a multiple of
// 64, at most 1024).  `sh` needs 17 ints.  Returns the exclusive prefix and
// stores the block total in *total.
__device__ __forceinline__ int block_excl_scan(int x, int *sh, int *total)
{
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    int incl = wave_incl_scan(x);
    if (lane == kWave - 1) sh[w] = incl;
    __syncthreads();
    if (threadIdx.x < kWave) {
        int v = threadIdx.x < nw ? sh[threadIdx.x] : 0;
        int vi = wave_incl_scan(v);
        if (threadIdx.x < nw) sh[threadIdx.x] = vi - v;
        if (threadIdx.x == kWave - 1) sh[16] = vi;
    }
    __syncthreads();
    int res = incl - x + sh[w];
    *total = sh[16];
    __syncthreads();
    return res;
}

}  // namespace wfd
