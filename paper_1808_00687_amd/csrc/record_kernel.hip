// Record kernel: back-pointers and raw lattice records of every token set,
// derived from the stored token sets after the search (token passing keeps a
// predecessor per token, Sec. 3 and Fig. 2; exact lattice generation keeps
// the arcs between surviving tokens, Sec. 1 and Sec. 3).
//
// Nothing here feeds the next frame of the search, so the frames of all
// utterances are processed in parallel: one block per (token set k,
// utterance).  A block
//   1. builds a hash table state -> survivor index of S_k in LDS;
//   2. goes through the epsilon arcs of the survivors of S_k (the first one
//      stored with the survivor by the search, the others from the graph):
//      an arc whose prefix cost is within the set's cutoff and whose
//      destination survived is an epsilon lattice arc, and the one that is
//      the destination's winning arc gives its back-pointer;
//   3. for k >= 1, goes through the candidates the search listed while it
//      expanded S_{k-1} (source survivor, arc, cost, destination): the same
//      for the emitting arcs into S_k.
// The start token's back-pointer is -1.  The search reserved each set's
// regions (one entry per emitting and per epsilon out-arc of the set); the
// block appends into them and stores the counts.  Sets larger than the LDS
// table are left to a second launch with a larger LDS table (or, beyond that,
// the utterance's device-memory table).
#include "device_util.h"

namespace wfd {

namespace {

constexpr int kRT = 1024;               // threads of a record block
constexpr int kRSlotBits = 13;
constexpr int kRSlots = 1 << kRSlotBits;
constexpr int kRFill = kRSlots / 4 * 3; // survivors per set the LDS table takes

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

// Back-pointers and records of token set k of utterance u, with the table t
// (cleared, of 2^(32 - t.shift) slots).
template <bool G>
__device__ void record_set(const Params &p, int u, int k, const RTab<G> &t, RSh &sh)
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
    const uint64_t *sv_tok = p.sv_tok + ly.sv0;
    int32_t *sv_prev = p.sv_prev + ly.sv0;

    // ---- 1. the table of S_k ----
    for (int i = tid; i < n; i += blockDim.x) rt_insert<G>(t, static_cast<uint32_t>(sv_state[b0 + i]), b0 + i);
    if (tid == 0) sh.nx = sh.ne = 0;
    __syncthreads();

    // ---- 2. the epsilon arcs of S_k ----
    // The winner of an epsilon-reached survivor is the arc whose candidate
    // equals the survivor's token: its cost is within the cutoff, so it is
    // among the arcs looked up here.
    const int64_t xbase = ly.lx0 + p.lx_off[ly.fo0 + k];
    for (int i0 = wid * kWave; i0 < n; i0 += nw * kWave) {
        const int i = i0 + lane;
        int xd = 0;
        float cst = 0.0f;
        int4 x = make_int4(0, 0, 0, 0);
        if (i < n) {
            const uint64_t tk = sv_tok[b0 + i];
            x = p.sv_x[ly.sv0 + b0 + i];
            cst = tok_cost(tk);
            xd = x.x;
            if (tok_arc(tk) < 0) sv_prev[b0 + i] = -1;   // the start token
        }
        // the first epsilon arc, stored with the survivor
        {
            bool rec = false;
            int4 r4 = make_int4(0, 0, 0, 0);
            const float pc = cst + __int_as_float(x.z);
            if (xd > 0 && okey(pc) <= cut) {
                const int32_t drel = rt_find<G>(t, static_cast<uint32_t>(x.y) & kDstMask);
                if (drel >= 0) {
                    if (tok_arc(sv_tok[drel]) == x.w) sv_prev[drel] = static_cast<int32_t>(b0 + i);
                    rec = p.lattice;
                    r4 = make_int4(static_cast<int>(b0 + i), drel, x.w, __float_as_int(pc));
                }
            }
            append(p.lat_x, xbase, &sh.nx, rec, r4);
        }
        // the others, from the epsilon rows, spread over the lanes
        const int xr = max(xd - 1, 0);
        const int incl = wave_incl_scan(xr);
        const int tot = __builtin_amdgcn_readlane(incl, kWave - 1);
        if (tot == 0) continue;
        int xb = 0;
        if (xr > 0) xb = p.g.srec[2 * static_cast<int64_t>(sv_state[b0 + i])].z + 1;
        const int pre = incl - xr;
        for (int q0 = 0; q0 < tot; q0 += kWave) {
            const int q = q0 + lane;
            const int o = owner_lane(pre, q);
            const int ob = __shfl(xb, o, kWave);
            const int op = __shfl(pre, o, kWave);
            const float oc = __shfl(cst, o, kWave);
            bool rec = false;
            int4 r4 = make_int4(0, 0, 0, 0);
            if (q < tot) {
                const int4 y = p.g.xarc[ob + (q - op)];
                const float pc = oc + __int_as_float(y.y);
                if (okey(pc) <= cut) {
                    const int32_t drel = rt_find<G>(t, static_cast<uint32_t>(y.x) & kDstMask);
                    if (drel >= 0) {
                        const int32_t src = static_cast<int32_t>(b0 + i0 + o);
                        if (tok_arc(sv_tok[drel]) == y.z) sv_prev[drel] = src;
                        rec = p.lattice;
                        r4 = make_int4(src, drel, y.z, __float_as_int(pc));
                    }
                }
            }
            append(p.lat_x, xbase, &sh.nx, rec, r4);
        }
    }

    // ---- 3. the candidates of S_{k-1}'s expansion into S_k ----
    if (k > 0) {
        const int64_t r0 = ly.le0 + p.le_off[ly.fo0 + k - 1];
        const int nc = static_cast<int>(p.cand_cnt[ly.fo0 + k - 1]);
        for (int c0 = wid * kWave; c0 < nc; c0 += nw * kWave) {
            const int c = c0 + lane;
            bool rec = false;
            int4 r4 = make_int4(0, 0, 0, 0);
            if (c < nc) {
                const int4 cd = p.cand[r0 + c];
                const int32_t drel = rt_find<G>(t, static_cast<uint32_t>(cd.w));
                if (drel >= 0) {
                    if (tok_arc(sv_tok[drel]) == cd.y) sv_prev[drel] = cd.x;
                    rec = p.lattice && okey(__int_as_float(cd.z)) <= cut;
                    r4 = make_int4(cd.x, drel, cd.y, cd.z);
                }
            }
            append(p.lat_e, r0, &sh.ne, rec, r4);
        }
    }
    __syncthreads();
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
    __shared__ RSh sh;
    const int k = blockIdx.x;
    const int u = blockIdx.y;
    UttState &st = p.st[u];
    if (st.status != 0 || k > st.Tp) return;
    const UttLayout &ly = p.lay[u];
    const int n = static_cast<int>(p.sv_off[ly.fo0 + k + 1] - p.sv_off[ly.fo0 + k]);
    if (n > min(kRFill, p.rec_fill)) {
        // left to the device-memory pass
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
    record_set<false>(p, u, k, t, sh);
}

// The sets too large for record_kernel's table: kLargeParts blocks per
// utterance share them (set k goes to part k mod kLargeParts); a set of up
// to kRBigFill survivors uses a 128 KB LDS table, a larger one the
// utterance's device-memory table (at most three quarters full: its size
// bounds the states a frame may reach), taken by part 0 alone.
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
                record_set<false>(p, u, kk, t, sh);
            } else {
                if (part != 0) continue;
                for (int64_t j = threadIdx.x; j < p.capG; j += blockDim.x) gt.keys[j] = kEmptyKey;
                __syncthreads();
                record_set<true>(p, u, kk, gt, sh);
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
