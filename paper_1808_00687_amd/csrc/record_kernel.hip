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
#include "record_set.h"

namespace wfd {

namespace {

// One block per (set k, utterance u) whose set fits the LDS table.
__global__ __launch_bounds__(kRT) void record_kernel(Params p)
{
    __shared__ uint32_t s_keys[kRSlots];
    __shared__ int32_t s_vals[kRSlots];
    __shared__ unsigned long long s_win[kRFill];
    __shared__ RSh sh;
    const int k = blockIdx.x;
    const int u = blockIdx.y;
    const UttState &st = p.st[u];
    if (st.status != 0 || k > st.Tp) return;
    record_one(p, u, k, s_keys, s_vals, s_win, sh);
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
                record_set<false, true>(p, u, kk, t, win, sh, lin_e(p, ly, kk), lin_x(p, ly, kk));
            } else {
                if (part != 0) continue;
                for (int64_t j = threadIdx.x; j < p.capG; j += blockDim.x) gt.keys[j] = kEmptyKey;
                __syncthreads();
                record_set<true, true>(p, u, kk, gt, win, sh, lin_e(p, ly, kk), lin_x(p, ly, kk));
            }
            __syncthreads();
        }
    }
}

// ---------------------------------------------------------------------------
// Incremental lattice pass beside the search (the paper runs lattice
// pruning on a stream of its own, concurrently with decoding, Sec. 3).
//
// One block per utterance follows the search: every stream_k token sets it
// records the finished sets (back-pointers, and raw lattice records into a
// ring) and prunes the raw records of the chunk against the frontier: with
// the extra cost of every token of the frontier set taken as 0, the backward
// pass gives each arc a lower bound of its final extra cost (every final
// extra cost is >= 0, and each step fl(fl(p - c) + e) is monotone in e),
// so an arc whose bound already exceeds the lattice beam is never kept, and
// removing it changes no kept arc's extra cost (a node with an extra cost
// within the beam keeps the out-arc that gives it).  The survivors are
// appended to the lattice regions, where the final pass (finish_kernel)
// prunes them exactly.  The raw records thus need a ring of a chunk's size
// instead of regions for the whole utterance.
// ---------------------------------------------------------------------------

constexpr long long kSpinLimit = 1LL << 30;   // polls of the progress count before giving up
struct LSh {
    RSh r;
    int prog;
    int cnt;
    int flag;
};

// Wait until the search has published at least `need` finished token sets
// (or failed: -1).  Thread 0 polls with relaxed loads (an acquire on every
// poll would invalidate the caches the searches on the same chiplet use);
// one acquire fence after the count is seen makes the sets visible.
// Returns the count, or -2 after the spin limit.
__device__ __forceinline__ int wait_sets(const Params &p, int u, int need, LSh &sh)
{
    if (threadIdx.x == 0) {
        int v = 0;
        for (long long i = 0;; i++) {
            v = __hip_atomic_load(p.prog + u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (v >= need || v < 0) break;
            if (i >= kSpinLimit) {
                v = -2;
                break;
            }
            __builtin_amdgcn_s_sleep(64);
        }
        sh.prog = v;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return sh.prog;
}

// Extra-cost lower bounds of the raw records of source sets [a, b) with the
// extra cost of every token of set b taken as 0 (the frontier), then the
// records within the lattice beam appended to the lattice regions.  With
// b > Tp (the last chunk) every record is kept for the final pass.
// Returns 0 or WFST_ECAPACITY.
__device__ int prune_chunk(const Params &p, int u, const UttLayout &ly, int a, int b, int Tp, LSh &sh, int64_t &ke,
                           int64_t &kx)
{
    const int tid = threadIdx.x;
    const int nt = blockDim.x;
    const int64_t *so = p.sv_off + ly.fo0;
    const uint32_t *key = p.sv_key + ly.sv0;
    uint32_t *eg = p.e_key + ly.sv0;
    const int4 *re = p.rng_e + u * p.rce;
    float *ree = p.rng_ee + u * p.rce;
    const int4 *rx = p.rng_x + u * p.rcx;
    float *rxe = p.rng_xe + u * p.rcx;
    const float lb = p.lattice_beam;
    const uint32_t kinf = okey(__int_as_float(0x7F800000));
    const bool last = b > Tp;
    if (!last) {
        for (int64_t i = so[b] + tid; i < so[b + 1]; i += nt) eg[i] = okey(0.0f);
        block_sync_vm();
        for (int j = b - 1; j >= a; j--) {
            for (int64_t i = so[j] + tid; i < so[j + 1]; i += nt) eg[i] = kinf;
            block_sync_vm();
            const int64_t e0 = p.rle_off[ly.fo0 + j], ne = p.le_cnt[ly.fo0 + j];
            for (int64_t r = tid; r < ne; r += nt) {
                const int64_t q = (e0 + r) % p.rce;
                const int4 x = re[q];
                const float d1 = __int_as_float(x.w) - okey_val(key[x.y]);
                const float ex = d1 + okey_val(ld_relaxed(eg + x.y));
                ree[q] = ex;
                atomicMin(eg + x.x, okey(ex));
            }
            block_sync_vm();
            const int64_t x0 = p.rlx_off[ly.fo0 + j], nx = p.lx_cnt[ly.fo0 + j];
            while (nx > 0) {
                if (tid == 0) sh.flag = 0;
                block_sync_vm();
                int changed = 0;
                for (int64_t r = tid; r < nx; r += nt) {
                    const int64_t q = (x0 + r) % p.rcx;
                    const int4 x = rx[q];
                    const float d1 = __int_as_float(x.w) - okey_val(key[x.y]);
                    const float ex = d1 + okey_val(ld_relaxed(eg + x.y));
                    rxe[q] = ex;
                    const uint32_t k = okey(ex);
                    if (k < ld_relaxed(eg + x.x)) {
                        atomicMin(eg + x.x, k);
                        changed = 1;
                    }
                }
                if (changed) sh.flag = 1;
                block_sync_vm();
                const int again = sh.flag;
                block_sync_vm();
                if (!again) break;
            }
        }
    }
    block_sync_vm();
    // the survivors of each source set, appended to the lattice regions
    for (int j = a; j < b && j <= Tp; j++) {
        for (int kind = 0; kind < 2; kind++) {
            const bool em = kind == 0;
            if (em && j == Tp) {
                if (tid == 0) {
                    p.le_off[ly.fo0 + j] = ke;
                    p.le_cnt[ly.fo0 + j] = 0;
                }
                continue;
            }
            const int64_t r0 = em ? p.rle_off[ly.fo0 + j] : p.rlx_off[ly.fo0 + j];
            const int64_t n = em ? p.le_cnt[ly.fo0 + j] : p.lx_cnt[ly.fo0 + j];
            const int64_t ring = em ? p.rce : p.rcx;
            const int4 *src = em ? re : rx;
            const float *sx = em ? ree : rxe;
            int4 *dst = em ? p.lat_e + ly.le0 : p.lat_x + ly.lx0;
            const int64_t cap = em ? ly.lecap : ly.lxcap;
            int64_t &fill = em ? ke : kx;
            if (tid == 0) sh.cnt = 0;
            block_sync_vm();
            for (int64_t r0i = 0; r0i < n; r0i += nt) {
                const int64_t r = r0i + tid;
                bool keep = false;
                int4 x = make_int4(0, 0, 0, 0);
                if (r < n) {
                    const int64_t q = (r0 + r) % ring;
                    x = src[q];
                    keep = last || sx[q] <= lb;
                }
                const uint64_t m = __ballot(keep);
                int bw = 0;
                if (m && lane_id() == 0) bw = atomicAdd(&sh.cnt, __popcll(m));
                bw = __builtin_amdgcn_readlane(bw, 0);
                if (keep) {
                    const int64_t at = fill + bw + rank_in(m);
                    if (at < cap) dst[at] = x;
                }
            }
            block_sync_vm();
            const int c = sh.cnt;
            block_sync_vm();
            if (fill + c > cap) return WFST_ECAPACITY;
            if (tid == 0) {
                if (em) {
                    p.le_off[ly.fo0 + j] = fill;
                    p.le_cnt[ly.fo0 + j] = c;
                } else {
                    p.lx_off[ly.fo0 + j] = fill;
                    p.lx_cnt[ly.fo0 + j] = c;
                }
            }
            fill += c;
        }
    }
    block_sync_vm();
    return 0;
}

__global__ __launch_bounds__(kRT) void lattice_stream_kernel(Params p)
{
    __shared__ uint32_t s_keys[kRSlots];
    __shared__ int32_t s_vals[kRSlots];
    __shared__ unsigned long long s_win[kRFill];
    __shared__ LSh sh;
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    const int Tp = st.Tp;   // from the classify kernel, before the search
    const UttLayout &ly = p.lay[u];
    const int64_t *so = p.sv_off + ly.fo0;
    const int64_t *rle = p.rle_off + ly.fo0;
    const int64_t *rlx = p.rlx_off + ly.fo0;
    const int K = p.stream_k;
    int4 *re = p.rng_e + u * p.rce;
    int4 *rx = p.rng_x + u * p.rcx;
    RTab<true> gt;
    const int64_t gbase = static_cast<int64_t>(u) * p.capG;
    gt.keys = p.rkeys + gbase;
    gt.vals = p.rvals + gbase;
    gt.mask = static_cast<uint32_t>(p.capG - 1);
    gt.shift = 32 - (31 - __clz(static_cast<int>(p.capG)));
    gt.mul = p.hash_mul;
    int64_t ke = 0, kx = 0;       // records kept in the lattice regions
    int rec = 0;                  // token sets recorded
    int prog = 0;
    int a = 0;                    // first source set not pruned yet
    int rc = 0;
    // A set's raw records sit in the rings at its reserved offsets (the
    // search reserves one slot per out-arc of the set), modulo the ring: the
    // emitting records of source set j from rle[j], its epsilon records from
    // rlx[j].  A chunk of source sets [a, b) and the epsilon records of set b
    // must fit the rings at once.
    while (a <= Tp) {
        const int bmax = min(a + K, Tp + 1);
        const int need = min(bmax, Tp) + 1;
        if (prog < need) {
            prog = wait_sets(p, u, need, sh);
            if (prog < 0) {
                rc = prog == -2 ? kStatusStreamTimeout : 0;
                break;
            }
        }
        // record sets up to bmax while the rings hold them: set k brings the
        // emitting records of source set k - 1 and the epsilon records of k
        int b = bmax;
        for (int k = rec; k <= min(bmax, Tp); k++) {
            if (rle[k] - rle[a] > p.rce || rlx[k + 1] - rlx[a] > p.rcx) {
                b = k - 1;
                break;
            }
            const int n = static_cast<int>(so[k + 1] - so[k]);
            const RecOut eo{re, k > 0 ? rle[k - 1] : 0, p.rce}, xo{rx, rlx[k], p.rcx};
            if (n <= min(kRFill, p.rec_fill)) {
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
                record_set<false, false>(p, u, k, t, s_win, sh.r, eo, xo);
            } else {
                for (int64_t j = threadIdx.x; j < p.capG; j += blockDim.x) gt.keys[j] = kEmptyKey;
                block_sync_vm();
                record_set<true, true>(p, u, k, gt, p.sv_win + ly.sv0 + so[k], sh.r, eo, xo);
            }
            rec = k + 1;
            __syncthreads();
        }
        if (b <= a) {
            rc = WFST_ECAPACITY;   // one token set does not fit the rings
            break;
        }
        rc = prune_chunk(p, u, ly, a, b, Tp, sh, ke, kx);
        if (rc) break;
        a = b;
    }
    if (rc && threadIdx.x == 0) set_status(st, rc);
    if (!rc && threadIdx.x == 0) st.lat_inc = ke + kx;
}

}  // namespace

hipError_t launch_lattice_stream(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(lattice_stream_kernel, dim3(p.U), dim3(kRT), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_record_large(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(record_large_kernel, dim3(p.U, kLargeParts), dim3(kRT), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_record(const Params &p, int max_frames, hipStream_t s)
{
    hipLaunchKernelGGL(record_kernel, dim3(max_frames + 1, p.U), dim3(kRT), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_record_large(p, s);
}

}  // namespace wfd
