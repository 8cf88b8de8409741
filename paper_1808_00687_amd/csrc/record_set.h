// Derivation of the back-pointers and lattice records of one token set
// (Sec. 3 predecessors, Sec. 1 and Sec. 3 exact lattices), shared by the
// record kernels and by the record workgroups that run beside the search.
// See record_kernel.hip for the method.
#pragma once

#include "device_util.h"

namespace wfd {

namespace {

constexpr int kRT = 1024;               // threads of a record block
constexpr int kRSlotBits = 13;
constexpr int kRSlots = 1 << kRSlotBits;
constexpr int kRFill = kRSlots / 4 * 3; // survivors per set the LDS table takes
constexpr unsigned long long kNoWin = ~0ull;

// state -> survivor index, open addressing with linear probing.  In device
// memory the table is touched by atomics in L2, so its loads bypass the CU
// cache.
template <bool G>
struct RTab {
    uint32_t *keys;
    int32_t *vals;
    uint32_t mask;
    int shift;   // 32 - log2(slots)
    uint32_t mul;   // hash multiplier
};

template <bool G, typename T>
__device__ __forceinline__ T rld(const T *ptr)
{
    if constexpr (G)
        return __hip_atomic_load(const_cast<T *>(ptr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
        return *ptr;
}

template <bool G>
__device__ __forceinline__ void rt_insert(const RTab<G> &t, uint32_t s, int32_t v)
{
    uint32_t h = hash_state(s, t.mul) >> t.shift;
    // survivor states are distinct: the first free slot on the probe path is s's
    while (atomicCAS(t.keys + h, kEmptyKey, s) != kEmptyKey) h = (h + 1) & t.mask;
    t.vals[h] = v;
}

template <bool G>
__device__ __forceinline__ int32_t rt_find(const RTab<G> &t, uint32_t s)
{
    uint32_t h = hash_state(s, t.mul) >> t.shift;
    for (uint32_t probe = 0; probe <= t.mask; probe++) {
        const uint32_t k = rld<G>(t.keys + h);
        if (k == s) return rld<G>(t.vals + h);
        if (k == kEmptyKey) return -1;
        h = (h + 1) & t.mask;
    }
    return -1;
}

// Where a set's records go: buf[base + i], or with ring > 0 the ring
// buf[(base + i) % ring] (base then counts records ever written to it).
struct RecOut {
    int4 *buf;
    int64_t base;
    int64_t ring;
};

// Append one record per lane (rec) at a block counter, one LDS add per
// wave.  The region or ring was reserved large enough.
__device__ __forceinline__ void append(const RecOut &o, int *cnt, bool rec, const int4 &r)
{
    const uint64_t m = __ballot(rec);
    if (!m) return;
    int b = 0;
    if (lane_id() == 0) b = atomicAdd(cnt, __popcll(m));
    b = __builtin_amdgcn_readlane(b, 0);
    if (rec) {
        const int64_t i = o.base + b + rank_in(m);
        o.buf[o.ring ? i % o.ring : i] = r;
    }
}

struct RSh {
    int nx, ne;   // records appended to the set's epsilon and emitting regions
};

// One arc into S_k per lane (valid): its candidate cost, user arc, source
// survivor and destination state.  A destination that survived gets a
// lattice record (returns true, when the lattice is on, with the record in
// r4) and, when the candidate ties the destination's cost, the arc competes
// for its back-pointer: the minimum of (user arc + 1) << 32 | source.
template <bool G>
__device__ __forceinline__ bool into_set(const Params &p, const RTab<G> &t, unsigned long long *win, int64_t b0,
                                         const uint32_t *sv_key, uint32_t cut, bool valid, float cand, int32_t arc,
                                         int32_t src, uint32_t dst, int4 &r4)
{
    bool rec = false;
    const uint32_t key = okey(cand);
    if (valid && key <= cut) {
        const int32_t drel = rt_find<G>(t, dst);
        if (drel >= 0) {
            if (sv_key[drel] == key) {
                const unsigned long long w =
                    (static_cast<unsigned long long>(static_cast<uint32_t>(arc) + 1u) << 32) | static_cast<uint32_t>(src);
                atomicMin(win + (drel - b0), w);
            }
            rec = p.lattice;
            r4 = make_int4(src, drel, arc, __float_as_int(cand));
        }
    }
    return rec;
}

// Back-pointers and records of token set k of utterance u, with the table t
// (cleared, of 2^(32 - t.shift) slots) and the winner array win (one entry
// per survivor of S_k: in LDS, or with GW in device memory).  The epsilon
// records of S_k go to xo, the emitting records into S_k (from S_{k-1}) to eo.
template <bool G, bool GW>
__device__ void record_set(const Params &p, int u, int k, const RTab<G> &t, unsigned long long *win, RSh &sh,
                           const RecOut &eo, const RecOut &xo)
{
    const UttLayout ly = p.lay[u];
    UttState &st = p.st[u];
    const int64_t *so = p.sv_off + ly.fo0;
    const int64_t b0 = so[k];
    const int n = static_cast<int>(so[k + 1] - b0);
    const uint32_t cut = p.cut_arr[ly.fo0 + k];
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wid = tid / kWave;
    const int nw = blockDim.x / kWave;
    const int32_t *sv_state = p.sv_state + ly.sv0;
    const uint32_t *sv_key = p.sv_key + ly.sv0;

    // ---- 1. the table of S_k, no winners yet ----
    for (int i = tid; i < n; i += blockDim.x) {
        rt_insert<G>(t, static_cast<uint32_t>(sv_state[b0 + i]), static_cast<int32_t>(b0 + i));
        win[i] = kNoWin;
    }
    if (tid == 0) sh.nx = sh.ne = 0;
    if constexpr (G || GW) vm_wait();
    __syncthreads();

    // ---- 2. the epsilon arcs of S_k ----
    for (int i0 = wid * kWave; i0 < n; i0 += nw * kWave) {
        const int i = i0 + lane;
        int xd = 0;
        float cst = 0.0f;
        int4 lo = make_int4(0, 0, 0, 0), x = make_int4(0, 0, 0, 0);
        if (i < n) {
            const int64_t s = sv_state[b0 + i];
            cst = okey_val(sv_key[b0 + i]);
            lo = p.g.srec[s];
            x = p.g.srec[s + 1];
            xd = lo.w - lo.z;
        }
        // the first epsilon arc, copied into the state record
        {
            int4 r4 = make_int4(0, 0, 0, 0);
            const bool rec = into_set<G>(p, t, win, b0, sv_key, cut, xd > 0, cst + __int_as_float(x.y), x.z,
                                         static_cast<int32_t>(b0 + i), static_cast<uint32_t>(x.x) & kDstMask, r4);
            append(xo, &sh.nx, rec, r4);
        }
        // the others, from the epsilon rows, spread over the lanes
        const int xr = max(xd - 1, 0);
        const int incl = wave_incl_scan(xr);
        const int tot = __builtin_amdgcn_readlane(incl, kWave - 1);
        if (tot == 0) continue;
        const int xb = lo.z + 1;
        const int pre = incl - xr;
        for (int q0 = 0; q0 < tot; q0 += kWave) {
            const int q = q0 + lane;
            const int o = owner_lane(pre, q);
            const int ob = __shfl(xb, o, kWave);
            const int op = __shfl(pre, o, kWave);
            const float oc = __shfl(cst, o, kWave);
            int4 y = make_int4(0, 0, 0, 0);
            if (q < tot) y = p.g.xarc[ob + (q - op)];
            int4 r4 = make_int4(0, 0, 0, 0);
            const bool rec = into_set<G>(p, t, win, b0, sv_key, cut, q < tot, oc + __int_as_float(y.y), y.z,
                                         static_cast<int32_t>(b0 + i0 + o), static_cast<uint32_t>(y.x) & kDstMask, r4);
            append(xo, &sh.nx, rec, r4);
        }
    }

    // ---- 3. the emitting arcs of S_{k-1}, expanded again into S_k ----
    if (k > 0) {
        const int64_t b1 = so[k - 1];
        const int n1 = static_cast<int>(b0 - b1);
        const int a1 = static_cast<int>(p.rle_off[ly.fo0 + k] - p.rle_off[ly.fo0 + k - 1]);
        const float *row = st.ll + static_cast<int64_t>(p.kept[ly.kept0 + k - 1]) * p.L;
        for (int i0 = wid * kWave; i0 < n1; i0 += nw * kWave) {
            const int i = i0 + lane;
            int deg = 0, eb = 0;
            float cst = 0.0f;
            if (i < n1) {
                const int pre_i = p.sv_epre[ly.sv0 + b1 + i];
                const int nxt = i + 1 < n1 ? p.sv_epre[ly.sv0 + b1 + i + 1] : a1;
                deg = nxt - pre_i;
                eb = p.sv_ebeg[ly.sv0 + b1 + i];
                cst = okey_val(sv_key[b1 + i]);
            }
            const int incl = wave_incl_scan(deg);
            const int tot = __builtin_amdgcn_readlane(incl, kWave - 1);
            const int pre = incl - deg;
            for (int q0 = 0; q0 < tot; q0 += kWave) {
                const int q = q0 + lane;
                const int o = owner_lane(pre, q);
                const int ob = __shfl(eb, o, kWave);
                const int op = __shfl(pre, o, kWave);
                const float oc = __shfl(cst, o, kWave);
                int4 y = make_int4(0, 0, 0, 0);
                int32_t ua = 0;
                float lv = 0.0f;
                if (q < tot) {
                    y = p.g.earc[ob + (q - op)];
                    ua = p.g.eua[ob + (q - op)];
                    lv = ldg(row + y.y);
                }
                const float t1 = oc + __int_as_float(y.z);
                int4 r4 = make_int4(0, 0, 0, 0);
                const bool rec = into_set<G>(p, t, win, b0, sv_key, cut, q < tot, t1 - lv, ua,
                                             static_cast<int32_t>(b1 + i0 + o), static_cast<uint32_t>(y.x) & kDstMask,
                                             r4);
                append(eo, &sh.ne, rec, r4);
            }
        }
    }
    // device-memory winners: every atomic complete before they are read back
    if constexpr (GW) vm_wait();
    __syncthreads();

    // ---- 4. back-pointers ----
    int bad = 0;
    for (int i = tid; i < n; i += blockDim.x) {
        unsigned long long w;
        if constexpr (GW) w = __hip_atomic_load(win + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else w = win[i];
        int32_t arc = -1, prev = -1;
        if (w != kNoWin) {
            arc = static_cast<int32_t>(static_cast<uint32_t>(w >> 32)) - 1;
            prev = static_cast<int32_t>(static_cast<uint32_t>(w));
        } else if (k != 0) {
            bad = 1;
        }
        p.sv_arc[ly.sv0 + b0 + i] = arc;
        p.sv_prev[ly.sv0 + b0 + i] = prev;
    }
    if (bad) set_status(st, kStatusNoBackPointer);
    if (tid == 0 && p.lattice) {
        p.lx_cnt[ly.fo0 + k] = sh.nx;
        if (k > 0) p.le_cnt[ly.fo0 + k - 1] = sh.ne;
        atomicAdd(reinterpret_cast<unsigned long long *>(&st.lx_cnt), static_cast<unsigned long long>(sh.nx));
        atomicAdd(reinterpret_cast<unsigned long long *>(&st.le_cnt), static_cast<unsigned long long>(sh.ne));
    }
}

// The lattice regions the search reserved for set k: emitting records into
// S_k (the region of S_{k-1}) and epsilon records of S_k.
__device__ __forceinline__ RecOut lin_e(const Params &p, const UttLayout &ly, int k)
{
    return RecOut{p.lat_e, k > 0 ? ly.le0 + p.rle_off[ly.fo0 + k - 1] : 0, 0};
}

__device__ __forceinline__ RecOut lin_x(const Params &p, const UttLayout &ly, int k)
{
    return RecOut{p.lat_x, ly.lx0 + p.rlx_off[ly.fo0 + k], 0};
}


// Token set k of utterance u with the LDS table s_keys/s_vals (kRSlots
// slots) and winners s_win (kRFill entries): sets larger than the table are
// left to the large-set pass.  Called by the whole block.
__device__ void record_one(const Params &p, int u, int k, uint32_t *s_keys, int32_t *s_vals,
                           unsigned long long *s_win, RSh &sh)
{
    UttState &st = p.st[u];
    const UttLayout &ly = p.lay[u];
    const int n = static_cast<int>(p.sv_off[ly.fo0 + k + 1] - p.sv_off[ly.fo0 + k]);
    if (n > min(kRFill, p.rec_fill)) {
        // left to the large-set pass
        if (threadIdx.x == 0) atomicOr(&st.big_sets, 1);
        return;
    }
    // a table of at least twice the set's size
    int bits = 10;
    while (bits < kRSlotBits && (1 << bits) < 2 * n) bits++;
    RTab<false> t;
    t.keys = s_keys;
    t.vals = s_vals;
    t.mask = (1u << bits) - 1u;
    t.shift = 32 - bits;
    t.mul = p.hash_mul;
    for (int i = threadIdx.x; i < (1 << bits); i += blockDim.x) s_keys[i] = kEmptyKey;
    __syncthreads();
    record_set<false, false>(p, u, k, t, s_win, sh, lin_e(p, ly, k), lin_x(p, ly, k));
}

}  // namespace

}  // namespace wfd
