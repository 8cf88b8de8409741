// Record kernel: back-pointers and raw lattice records of every token set,
// derived from the stored token sets after the search (token passing keeps a
// predecessor per token, Sec. 3 and Fig. 2; exact lattice generation keeps
// the arcs between surviving tokens, Sec. 1 and Sec. 3).
//
// Nothing here feeds the next frame of the search, so the frames of all
// utterances are processed in parallel: one block per (token set k,
// utterance).  A block
//   1. builds a hash table state -> survivor index of S_k in LDS;
//   2. goes through the epsilon arcs of the survivors of S_k (rows from the
//      state records of the graph): an arc whose candidate cost c(s) + w is
//      within the set's cutoff and whose destination survived is an epsilon
//      lattice arc;
//   3. for k >= 1, expands the emitting arcs of S_{k-1} again with the
//      frame's log-likelihoods, (c(s) + w) - ll, the same arithmetic as the
//      search: a candidate within the cutoff of S_k whose destination
//      survived is an emitting lattice arc;
//   4. gives each survivor of S_k its back-pointer: among the arcs of steps
//      2 and 3 whose candidate cost key equals the survivor's cost key, the
//      lowest user arc (and its source survivor).  That is the arc a minimum
//      over (cost, arc) pairs keeps, so the token is the one recombination
//      with the arc tie-break defines.  Every such arc is seen: its cost is
//      the survivor's, within the cutoff, and its source survived (epsilon
//      weights are >= 0 and pruning keeps every tie, so a source is never
//      above its destination).  The start token of S_0 has no such arc.
// The search reserved each set's regions (one entry per emitting and per
// epsilon out-arc of the set); the block appends into them and stores the
// counts.  Sets larger than the LDS table are left to a second launch with a
// larger LDS table (or, beyond that, the utterance's device-memory table).
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

// Append one record per lane (rec) at base + a block counter, one LDS add per
// wave.  The region was reserved large enough by the search.
__device__ __forceinline__ void append(int4 *buf, int64_t base, int *cnt, bool rec, const int4 &r)
{
    const uint64_t m = __ballot(rec);
    if (!m) return;
    int b = 0;
    if (lane_id() == 0) b = atomicAdd(cnt, __popcll(m));
    b = __builtin_amdgcn_readlane(b, 0);
    if (rec) buf[base + b + rank_in(m)] = r;
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
// per survivor of S_k: in LDS, or with GW in device memory).
template <bool G, bool GW>
__device__ void record_set(const Params &p, int u, int k, const RTab<G> &t, unsigned long long *win, RSh &sh)
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
    __syncthreads();

    // ---- 2. the epsilon arcs of S_k ----
    const int64_t xbase = ly.lx0 + p.lx_off[ly.fo0 + k];
    for (int i0 = wid * kWave; i0 < n; i0 += nw * kWave) {
        const int i = i0 + lane;
        int xd = 0;
        float cst = 0.0f;
        int4 lo = make_int4(0, 0, 0, 0), x = make_int4(0, 0, 0, 0);
        if (i < n) {
            const int64_t s = sv_state[b0 + i];
            cst = okey_val(sv_key[b0 + i]);
            lo = p.g.srec[2 * s];
            x = p.g.srec[2 * s + 1];
            xd = lo.w - lo.z;
        }
        // the first epsilon arc, copied into the state record
        {
            int4 r4 = make_int4(0, 0, 0, 0);
            const bool rec = into_set<G>(p, t, win, b0, sv_key, cut, xd > 0, cst + __int_as_float(x.y), x.z,
                                         static_cast<int32_t>(b0 + i), static_cast<uint32_t>(x.x) & kDstMask, r4);
            append(p.lat_x, xbase, &sh.nx, rec, r4);
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
            append(p.lat_x, xbase, &sh.nx, rec, r4);
        }
    }

    // ---- 3. the emitting arcs of S_{k-1}, expanded again into S_k ----
    if (k > 0) {
        const int64_t b1 = so[k - 1];
        const int n1 = static_cast<int>(b0 - b1);
        const int64_t r0 = ly.le0 + p.le_off[ly.fo0 + k - 1];
        const int a1 = static_cast<int>(p.le_off[ly.fo0 + k] - p.le_off[ly.fo0 + k - 1]);
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
                float lv = 0.0f;
                if (q < tot) {
                    y = p.g.earc[ob + (q - op)];
                    lv = ldg(row + y.y);
                }
                const float t1 = oc + __int_as_float(y.z);
                int4 r4 = make_int4(0, 0, 0, 0);
                const bool rec = into_set<G>(p, t, win, b0, sv_key, cut, q < tot, t1 - lv, y.w,
                                             static_cast<int32_t>(b1 + i0 + o), static_cast<uint32_t>(y.x) & kDstMask,
                                             r4);
                append(p.lat_e, r0, &sh.ne, rec, r4);
            }
        }
    }
    // device-memory winners: every atomic complete before they are read back
    if constexpr (GW) __threadfence();
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

// One block per (set k, utterance u) whose set fits the LDS table.
__global__ __launch_bounds__(kRT) void record_kernel(Params p)
{
    __shared__ uint32_t s_keys[kRSlots];
    __shared__ int32_t s_vals[kRSlots];
    __shared__ unsigned long long s_win[kRFill];
    __shared__ RSh sh;
    const int k = blockIdx.x;
    const int u = blockIdx.y;
    UttState &st = p.st[u];
    if (st.status != 0 || k > st.Tp) return;
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
    record_set<false, false>(p, u, k, t, s_win, sh);
}

// The sets too large for record_kernel's table: kLargeParts blocks per
// utterance share them (set k goes to part k mod kLargeParts); a set of up
// to kRBigFill survivors uses a 128 KB LDS table, a larger one the
// utterance's device-memory table (at most three quarters full: its size
// bounds the states a frame may reach), taken by part 0 alone.  Their
// back-pointer winners are kept in device memory.
constexpr int kLargeParts = 8;
constexpr int kRBigBits = 14;
constexpr int kRBigFill = (1 << kRBigBits) / 4 * 3;

__global__ __launch_bounds__(kRT) void record_large_kernel(Params p)
{
    __shared__ uint32_t s_keys[1 << kRBigBits];
    __shared__ int32_t s_vals[1 << kRBigBits];
    __shared__ RSh sh;
    __shared__ int s_list[kRT];
    __shared__ int s_n;
    const int u = blockIdx.x;
    const int part = blockIdx.y;
    const UttState &st = p.st[u];
    if (st.status != 0 || !st.big_sets) return;
    const UttLayout &ly = p.lay[u];
    RTab<true> gt;
    const int64_t gbase = static_cast<int64_t>(u) * p.capG;
    gt.keys = p.gkeys + gbase;
    gt.vals = p.gslots + gbase;
    gt.mask = static_cast<uint32_t>(p.capG - 1);
    gt.shift = 32 - (31 - __clz(static_cast<int>(p.capG)));
    gt.mul = p.hash_mul;
    const int big_fill = min(kRBigFill, p.rec_big_fill);
    // the large sets, kRT frames at a time
    for (int k0 = 0; k0 <= st.Tp; k0 += kRT) {
        if (threadIdx.x == 0) s_n = 0;
        __syncthreads();
        const int k = k0 + threadIdx.x;
        if (k <= st.Tp && p.sv_off[ly.fo0 + k + 1] - p.sv_off[ly.fo0 + k] > min(kRFill, p.rec_fill))
            s_list[atomicAdd(&s_n, 1)] = k;
        __syncthreads();
        const int nl = s_n;
        for (int i = 0; i < nl; i++) {
            const int kk = s_list[i];
            unsigned long long *win = p.sv_win + ly.sv0 + p.sv_off[ly.fo0 + kk];
            const int n = static_cast<int>(p.sv_off[ly.fo0 + kk + 1] - p.sv_off[ly.fo0 + kk]);
            if (n <= big_fill) {
                if (kk % kLargeParts != part) continue;
                int bits = 10;
                while (bits < kRBigBits && (1 << bits) < 2 * n) bits++;
                RTab<false> t;
                t.keys = s_keys;
                t.vals = s_vals;
                t.mask = (1u << bits) - 1u;
                t.shift = 32 - bits;
                t.mul = p.hash_mul;
                for (int j = threadIdx.x; j < (1 << bits); j += blockDim.x) s_keys[j] = kEmptyKey;
                __syncthreads();
                record_set<false, true>(p, u, kk, t, win, sh);
            } else {
                if (part != 0) continue;
                for (int64_t j = threadIdx.x; j < p.capG; j += blockDim.x) gt.keys[j] = kEmptyKey;
                __syncthreads();
                record_set<true, true>(p, u, kk, gt, win, sh);
            }
            __syncthreads();
        }
    }
}

}  // namespace

hipError_t launch_record(const Params &p, int max_frames, hipStream_t s)
{
    hipLaunchKernelGGL(record_kernel, dim3(max_frames + 1, p.U), dim3(kRT), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(record_large_kernel, dim3(p.U, kLargeParts), dim3(kRT), 0, s, p);
    return hipGetLastError();
}

}  // namespace wfd
