// End-of-utterance kernels: finalTransition and backtrace (Alg. 1 of the
// paper), lattice-beam pruning of the recorded lattice (the backward pass of
// exact lattice generation, Sec. 1 and Sec. 3), and the sorted lattice output.
#include <algorithm>

#include "device_util.h"

namespace wfd {

namespace {

// finalTransition: tot(s) = fl(c(s) + f(s)) over the last token set; the best
// is the smallest (cost key, state).  If final costs are given but no final
// state is active, every state counts as final with cost 0.
__global__ __launch_bounds__(256) void final_kernel(Params p)
{
    __shared__ uint64_t sh_min[4];
    __shared__ int sh_fallback;
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    if (st.status != 0) return;
    const UttLayout &ly = p.lay[u];
    const int Tp = st.Tp;
    const int64_t a = p.sv_off[ly.fo0 + Tp], b = p.sv_off[ly.fo0 + Tp + 1];
    const uint32_t kinf = okey(__int_as_float(0x7F800000));
    uint64_t best = ~0ull;
    for (int pass = 0; pass < 2; pass++) {
        const bool use_final = p.g.final_w != nullptr && pass == 0;
        uint64_t m = ~0ull;
        for (int64_t i = a + threadIdx.x; i < b; i += blockDim.x) {
            int s = p.sv_state[ly.sv0 + i];
            float c = okey_val(p.sv_key[ly.sv0 + i]);
            float f = use_final ? p.g.final_w[s] : 0.0f;
            float tot = c + f;
            uint64_t v = (static_cast<uint64_t>(okey(tot)) << 32) | static_cast<uint32_t>(s);
            m = v < m ? v : m;
        }
        m = wave_min_u64(m);
        if (lane_id() == 0) sh_min[threadIdx.x / kWave] = m;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint64_t x = sh_min[0];
            for (int w = 1; w < 4; w++) x = sh_min[w] < x ? sh_min[w] : x;
            sh_min[0] = x;
            sh_fallback = use_final && static_cast<uint32_t>(x >> 32) >= kinf;
        }
        __syncthreads();
        best = sh_min[0];
        const int fb = sh_fallback;
        __syncthreads();
        if (pass == 0 && fb) continue;
        if (threadIdx.x == 0) {
            st.reached_final = (pass == 0) ? 1 : 0;
            st.final_state = static_cast<int32_t>(static_cast<uint32_t>(best));
            st.final_cost = okey_val(static_cast<uint32_t>(best >> 32));
        }
        break;
    }
    const int bs = static_cast<int32_t>(static_cast<uint32_t>(best));
    for (int64_t i = a + threadIdx.x; i < b; i += blockDim.x)
        if (p.sv_state[ly.sv0 + i] == bs) st.final_sv = static_cast<int32_t>(i);
}

// backtrace (Alg. 1), one block per utterance.  Lane 0 follows the
// survivor back-pointers from the final token, one dependent load per step,
// and lists the survivors of the path; then the whole block turns them into
// arcs and original frame indices (an emitting arc of decoded frame j lies
// in frame kept[j - 1]; epsilon arcs have frame -1).  The path is written at
// the end of the utterance's path region, last arc last.
__device__ void backtrace_block(const Params &p, int u, int *sh)
{
    UttState &st = p.st[u];
    const UttLayout &ly = p.lay[u];
    const int64_t end = ly.path0 + ly.pathcap;
    if (threadIdx.x == 0) {
        int64_t i = st.final_sv;
        int cnt = 0;
        while (true) {
            const int a = p.sv_arc[ly.sv0 + i];
            const int prev = p.sv_prev[ly.sv0 + i];
            if (a < 0) break;
            if (cnt >= ly.pathcap || prev < 0) {
                set_status(st, WFST_ECAPACITY);
                break;
            }
            p.path_arc[end - 1 - cnt] = static_cast<int32_t>(i);
            cnt++;
            i = prev;
        }
        sh[0] = cnt;
    }
    __syncthreads();
    const int cnt = sh[0];
    const int Tp = st.Tp;
    // entry k counts from the final token backwards; its decoded frame is
    // Tp minus the emitting arcs of entries 0 .. k - 1
    int carry = 0;
    for (int k0 = 0; k0 < cnt; k0 += blockDim.x) {
        const int k = k0 + threadIdx.x;
        int a = -1;
        bool emit = false;
        if (k < cnt) {
            const int64_t i = p.path_arc[end - 1 - k];
            a = p.sv_arc[ly.sv0 + i];
            emit = p.g.arc_src[a] >= 0;
        }
        int total;
        const int before = carry + block_excl_scan(emit ? 1 : 0, sh + 1, &total);
        if (k < cnt) {
            int fr = -1;
            if (emit) {
                const int j = Tp - before;
                if (j >= 1) fr = p.kept[ly.kept0 + j - 1];
                else set_status(st, WFST_ECAPACITY);
            }
            p.path_arc[end - 1 - k] = a;
            p.path_frame[end - 1 - k] = fr;
        }
        carry += total;
    }
    if (threadIdx.x == 0) st.path_len = cnt;
}

// s_waitcnt immediate: vmcnt(0), the other counters left free
constexpr int kWaitVm0 = 0x0F70;
constexpr int kLatLds = 8192;   // survivors per token set kept in LDS by the backward pass
constexpr int kLatT = 1024;     // threads of a finish block
constexpr int kRE = 1;          // emitting records per thread held in registers
constexpr int kRX = 1;          // epsilon records per thread held in registers
constexpr int kRC = 1;          // survivors per thread held in registers

// Where the records and survivors of one token set j lie.
struct LatMeta {
    int64_t b0, nB;   // S_j
    int64_t e0, e1;   // emitting records (source in S_j, destination in S_j+1)
    int64_t x0, x1;   // epsilon records (both ends in S_j)
};

// Inputs of one token set, loaded a set ahead of their use.
struct LatRegs {
    int4 e[kRE];
    int4 x[kRX];
    uint32_t t[kRC];   // cost keys
};

__device__ __forceinline__ LatMeta lat_meta(const Params &p, const UttLayout &ly, int j, int Tp)
{
    LatMeta m;
    const int64_t *so = p.sv_off + ly.fo0;
    m.b0 = so[j];
    m.nB = so[j + 1] - so[j];
    m.e0 = j < Tp ? p.le_off[ly.fo0 + j] : 0;
    m.e1 = j < Tp ? m.e0 + p.le_cnt[ly.fo0 + j] : 0;
    m.x0 = p.lx_off[ly.fo0 + j];
    m.x1 = m.x0 + p.lx_cnt[ly.fo0 + j];
    return m;
}

// The same offsets loaded by lanes 0-5 of each wave with vector loads, to be
// unpacked a step later: a scalar load would be waited for at the next LDS
// barrier (scalar loads and LDS share one wait counter), a vector load only
// where its value is used.
__device__ __forceinline__ int64_t lat_meta_issue(const Params &p, const UttLayout &ly, int j, int Tp)
{
    const int l = lane_id();
    const int64_t f = ly.fo0 + j;
    const int64_t *a = nullptr;
    if (l == 0) a = p.sv_off + f;
    else if (l == 1) a = p.sv_off + f + 1;
    else if (l == 2 && j < Tp) a = p.le_off + f;
    else if (l == 3 && j < Tp) a = p.le_cnt + f;
    else if (l == 4) a = p.lx_off + f;
    else if (l == 5) a = p.lx_cnt + f;
    return a ? *a : 0;
}

__device__ __forceinline__ int64_t lane64(int64_t v, int l)
{
    const int lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint64_t>(v)), l);
    const int hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint64_t>(v) >> 32), l);
    return static_cast<int64_t>((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo));
}

__device__ __forceinline__ LatMeta lat_meta_take(int64_t v)
{
    LatMeta m;
    m.b0 = lane64(v, 0);
    m.nB = lane64(v, 1) - m.b0;
    m.e0 = lane64(v, 2);
    m.e1 = m.e0 + lane64(v, 3);
    m.x0 = lane64(v, 4);
    m.x1 = m.x0 + lane64(v, 5);
    return m;
}

// What a step of the backward pass leaves to be stored at the start of the
// next: the extra costs of its register-held records and its kept count.
struct LatPend {
    float ee[kRE];
    float ex[kRX];
    int64_t e0, e1, x0, x1;
    unsigned long long kept;
    int j;
};

__device__ __forceinline__ void lat_flush(const Params &p, const UttLayout &ly, LatPend &pd,
                                          unsigned long long *kcnt)
{
    const int tid = threadIdx.x;
#pragma unroll
    for (int q = 0; q < kRE; q++) {
        const int64_t r = pd.e0 + tid + q * kLatT;
        if (r < pd.e1) p.ex_e[ly.le0 + r] = pd.ee[q];
    }
#pragma unroll
    for (int q = 0; q < kRX; q++) {
        const int64_t r = pd.x0 + tid + q * kLatT;
        if (r < pd.x1) p.ex_x[ly.lx0 + r] = pd.ex[q];
    }
    if (pd.j >= 0) {
        // a thread keeps fewer than 2^31 arcs of one set
        const int k = __builtin_amdgcn_readlane(wave_incl_scan(static_cast<int>(pd.kept)), kWave - 1);
        if (lane_id() == 0 && k) atomicAdd(kcnt + pd.j, static_cast<unsigned long long>(k));
    }
    pd.e0 = pd.e1 = pd.x0 = pd.x1 = 0;
    pd.j = -1;
    pd.kept = 0;
}

__device__ __forceinline__ void lat_fetch(const Params &p, const UttLayout &ly, const LatMeta &m, LatRegs &r)
{
    const int tid = threadIdx.x;
#pragma unroll
    for (int q = 0; q < kRE; q++) {
        const int64_t i = m.e0 + tid + q * kLatT;
        r.e[q] = i < m.e1 ? p.lat_e[ly.le0 + i] : make_int4(0, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < kRX; q++) {
        const int64_t i = m.x0 + tid + q * kLatT;
        r.x[q] = i < m.x1 ? p.lat_x[ly.lx0 + i] : make_int4(0, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < kRC; q++) {
        const int64_t i = tid + q * kLatT;
        r.t[q] = i < m.nB ? p.sv_key[ly.sv0 + m.b0 + i] : kEmptyKey;
    }
}

// Lattice-beam pruning, one block per utterance, token sets from last to
// first.  e(j, s) is the extra cost of the best completion from node (j, s):
// at the last set e = fl(tot(s) - B); an arc from (j, s) with prefix cost p
// into (j', d) has ex = fl(fl(p - c_j'(d)) + e(j', d)), and e(j, s) is the
// minimum ex over its recorded out-arcs.  Epsilon arcs inside a set are
// iterated to their fixed point (the epsilon graph is acyclic).
//
// The costs and extra costs of S_j and S_j+1 live in LDS and the records of
// a set in registers, loaded while the previous set is processed; a set
// larger than kLatLds is processed in device memory instead.  Kept arcs are
// counted per set into lo_off (zeroed by the host), then turned into output
// offsets.
__device__ void lattice_sets(const Params &p, int u, uint32_t *s_e, float *s_c, int *sh)
{
    UttState &st = p.st[u];
    const UttLayout ly = p.lay[u];
    const int tid = threadIdx.x;
    const int Tp = st.Tp;
    const float lb = p.lattice_beam;
    const float B = st.final_cost;
    const bool use_final = p.g.final_w != nullptr && st.reached_final;
    uint32_t *eg = p.e_key + ly.sv0;
    const uint32_t *tok = p.sv_key + ly.sv0;   // cost keys
    const int64_t *so = p.sv_off + ly.fo0;
    unsigned long long *kcnt = reinterpret_cast<unsigned long long *>(p.lo_off + ly.fo0);
    const uint32_t kinf = okey(__int_as_float(0x7F800000));
    int *flag = sh;   // three rotating "changed" flags of the epsilon rounds
    int hA = 0;          // LDS half holding S_j+1
    bool a_lds = false;  // S_j+1's costs and extra costs are in that half
    // Two-deep pipeline: while set j is processed, the records of set j-1
    // are in flight (loaded into the second register set) and so are the
    // offsets of set j-2.  The extra costs of the register-held records are
    // stored at the start of the next step, after the prefetched registers
    // have been taken over: a wait for a load also waits for every store
    // issued after it, so stores at the end of a step would stall the next.
    LatMeta mc = lat_meta(p, ly, Tp, Tp);
    LatMeta mn{};
    if (Tp > 0) mn = lat_meta(p, ly, Tp - 1, Tp);
    LatRegs cur, nxt;
    lat_fetch(p, ly, mc, cur);
    LatPend pd;
    pd.e0 = pd.e1 = pd.x0 = pd.x1 = 0;
    pd.j = -1;
    pd.kept = 0;
    int64_t a0 = so[Tp + 1], nA = 0;   // S_j+1
    bool b_ready = false;              // S_j's extra costs are initialised in LDS
    const int64_t lcap = min(kLatLds, p.lat_lds);
    for (int j = Tp; j >= 0; j--) {
        // Everything the last step loaded has arrived (it was issued a step
        // ago).  Waiting for it here, before this step issues its own loads,
        // tells the compiler so: otherwise its first use of the current set
        // would wait for the loads issued below as well.
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        if (j > 0) lat_fetch(p, ly, mn, nxt);
        const int64_t mv2 = j > 1 ? lat_meta_issue(p, ly, j - 2, Tp) : 0;
        lat_flush(p, ly, pd, kcnt);
        const bool g = mc.nB > lcap || nA > lcap;
        const int hB = hA ^ 1;
        uint32_t *eA = s_e + hA * kLatLds, *eB = s_e + hB * kLatLds;
        float *cA = s_c + hA * kLatLds, *cB = s_c + hB * kLatLds;
        const int64_t b0 = mc.b0, nB = mc.nB;
        unsigned long long kept = 0;
        if (!g) {
            // ---- S_j and S_j+1 in LDS, records in registers ----
            if (tid == 0) flag[0] = 0;
#pragma unroll
            for (int q = 0; q < kRC; q++) {
                const int64_t i = tid + q * kLatT;
                if (i < nB) cB[i] = okey_val(cur.t[q]);
            }
            for (int64_t i = tid + kRC * kLatT; i < nB; i += kLatT) cB[i] = okey_val(tok[b0 + i]);
            // The costs of S_j are first read after the next barrier; its
            // extra costs were set to +inf by the previous step unless that
            // step ran in device memory (or this is the last set).
            if (!b_ready) {
                if (j == Tp) {
                    for (int64_t i = tid; i < nB; i += kLatT) {
                        const float c = okey_val(tok[b0 + i]);
                        const float f = use_final ? p.g.final_w[p.sv_state[ly.sv0 + b0 + i]] : 0.0f;
                        eB[i] = okey((c + f) - B);
                    }
                } else {
                    for (int64_t i = tid; i < nB; i += kLatT) eB[i] = kinf;
                }
            }
            if (!a_lds) {
                // S_j+1 was processed in device memory: bring it into LDS
                for (int64_t i = tid; i < nA; i += kLatT) {
                    eA[i] = ld_relaxed(eg + a0 + i);
                    cA[i] = okey_val(tok[a0 + i]);
                }
            }
            if (!b_ready || !a_lds) lds_barrier();
            // emitting arcs into S_j+1
#pragma unroll
            for (int q = 0; q < kRE; q++) {
                const int64_t r = mc.e0 + tid + q * kLatT;
                pd.ee[q] = 0.0f;
                if (r < mc.e1) {
                    const int4 x = cur.e[q];
                    const float d1 = __int_as_float(x.w) - cA[x.y - a0];
                    const float ex = d1 + okey_val(eA[x.y - a0]);
                    pd.ee[q] = ex;
                    atomicMin(eB + (x.x - b0), okey(ex));
                    kept += ex <= lb;
                }
            }
            pd.e0 = mc.e0;
            pd.e1 = mc.e1;
            for (int64_t r = mc.e0 + tid + kRE * kLatT; r < mc.e1; r += kLatT) {
                const int4 x = p.lat_e[ly.le0 + r];
                const float d1 = __int_as_float(x.w) - cA[x.y - a0];
                const float ex = d1 + okey_val(eA[x.y - a0]);
                p.ex_e[ly.le0 + r] = ex;
                atomicMin(eB + (x.x - b0), okey(ex));
                kept += ex <= lb;
            }
            lds_barrier();
            // S_j+1 is no longer read: its half takes the extra costs of
            // S_j-1, +inf until the next step's arcs lower them
            const bool next_lds = j > 0 && mn.nB <= lcap && nB <= lcap;
            if (next_lds)
                for (int64_t i = tid; i < mn.nB; i += kLatT) eA[i] = kinf;
            if (mc.x1 > mc.x0) {
                float exr[kRX];
                unsigned long long kx = 0;
                for (int it = 0;; it++) {
                    if (tid == 0) flag[(it + 1) % 3] = 0;
                    int changed = 0;
                    kx = 0;
#pragma unroll
                    for (int q = 0; q < kRX; q++) {
                        const int64_t r = mc.x0 + tid + q * kLatT;
                        exr[q] = 0.0f;
                        if (r < mc.x1) {
                            const int4 x = cur.x[q];
                            const float d1 = __int_as_float(x.w) - cB[x.y - b0];
                            const float ex = d1 + okey_val(eB[x.y - b0]);
                            exr[q] = ex;
                            const uint32_t k = okey(ex);
                            if (k < eB[x.x - b0]) {
                                atomicMin(eB + (x.x - b0), k);
                                changed = 1;
                            }
                            kx += ex <= lb;
                        }
                    }
                    for (int64_t r = mc.x0 + tid + kRX * kLatT; r < mc.x1; r += kLatT) {
                        const int4 x = p.lat_x[ly.lx0 + r];
                        const float d1 = __int_as_float(x.w) - cB[x.y - b0];
                        const float ex = d1 + okey_val(eB[x.y - b0]);
                        p.ex_x[ly.lx0 + r] = ex;
                        const uint32_t k = okey(ex);
                        if (k < eB[x.x - b0]) {
                            atomicMin(eB + (x.x - b0), k);
                            changed = 1;
                        }
                        kx += ex <= lb;
                    }
                    if (changed) flag[it % 3] = 1;
                    lds_barrier();
                    if (!flag[it % 3]) break;
                }
                // the last round changed nothing: its extra costs are final
#pragma unroll
                for (int q = 0; q < kRX; q++) pd.ex[q] = exr[q];
                pd.x0 = mc.x0;
                pd.x1 = mc.x1;
                kept += kx;
            }
            // the epsilon rounds' barriers publish that initialisation;
            // without rounds one barrier does
            if (next_lds && mc.x1 <= mc.x0) lds_barrier();
            b_ready = next_lds;
            // a following set processed in device memory reads S_j there
            const bool next_g = j > 0 && (mn.nB > lcap || nB > lcap);
            if (next_g)
                for (int64_t i = tid; i < nB; i += kLatT) eg[b0 + i] = eB[i];
        } else {
            // ---- a set larger than the LDS arrays: device memory ----
            b_ready = false;
            for (int64_t i = tid; i < nB; i += kLatT) {
                uint32_t e0 = kinf;
                if (j == Tp) {
                    const float c = okey_val(tok[b0 + i]);
                    const float f = use_final ? p.g.final_w[p.sv_state[ly.sv0 + b0 + i]] : 0.0f;
                    e0 = okey((c + f) - B);
                }
                eg[b0 + i] = e0;
            }
            __syncthreads();
            for (int64_t r = mc.e0 + tid; r < mc.e1; r += kLatT) {
                const int4 x = p.lat_e[ly.le0 + r];
                const float d1 = __int_as_float(x.w) - okey_val(tok[x.y]);
                const float ex = d1 + okey_val(ld_relaxed(eg + x.y));
                p.ex_e[ly.le0 + r] = ex;
                atomicMin(eg + x.x, okey(ex));
                kept += ex <= lb;
            }
            __syncthreads();
            if (mc.x1 > mc.x0) {
                unsigned long long kx = 0;
                while (true) {
                    if (tid == 0) flag[0] = 0;
                    __syncthreads();
                    int changed = 0;
                    kx = 0;
                    for (int64_t r = mc.x0 + tid; r < mc.x1; r += kLatT) {
                        const int4 x = p.lat_x[ly.lx0 + r];
                        const float d1 = __int_as_float(x.w) - okey_val(tok[x.y]);
                        const float ex = d1 + okey_val(ld_relaxed(eg + x.y));
                        p.ex_x[ly.lx0 + r] = ex;
                        const uint32_t k = okey(ex);
                        if (k < ld_relaxed(eg + x.x)) {
                            atomicMin(eg + x.x, k);
                            changed = 1;
                        }
                        kx += ex <= lb;
                    }
                    if (changed) flag[0] = 1;
                    __syncthreads();
                    const int again = flag[0];
                    __syncthreads();
                    if (!again) break;
                }
                kept += kx;
            }
        }
        pd.kept = kept;
        pd.j = j;
        a0 = b0;
        nA = nB;
        hA = hB;
        a_lds = !g;
        if (j > 0) cur = nxt;
        mc = mn;
        mn = j > 1 ? lat_meta_take(mv2) : LatMeta{};
    }
    lat_flush(p, ly, pd, kcnt);
}

// ---------------------------------------------------------------------------
// The backward pass of an utterance whose token sets all hold at most
// kSmallSet survivors, emitting records and epsilon records (the CTC-style
// configurations).  The block pass spends a set's time mostly on its waves'
// bookkeeping and barriers, whatever the set's size.  Here one wave
// (wave 0) computes the nodes' extra costs set after set from LDS alone,
// while the block's other waves load the coming sets into a ring of LDS
// slots; each slot is handed over with a workgroup-scope flag, filled after
// the previous set in it has been consumed.  Then the whole block derives
// every record's extra cost from its destination's, and the kept counts, set
// by set in parallel.  The arithmetic is the block pass's, step for step, so
// the extra costs, the kept arcs and their order are the same bit for bit.
// Every wait is bounded: a pass that stops hearing from the other side
// reports an error instead of hanging.
// ---------------------------------------------------------------------------
constexpr int kSmallSet = 64;                 // survivors and records per set (one per lane)
constexpr int kRing = 16;                     // sets in flight between the loading waves and wave 0
constexpr long long kSmallSpin = 1LL << 24;   // polls of one flag before a pass gives up (unless lat_spin sets it)

struct SmallSlot {
    int b0;                   // the set's first survivor (utterance-relative)
    int nB, ne, nx;           // survivors, emitting records (into the next set), epsilon records
    uint32_t key[kSmallSet];  // survivors' cost keys
    int es[kSmallSet];        // emitting records: source survivor (this set),
    int ed[kSmallSet];        // destination survivor (the next set)
    uint32_t ep[kSmallSet];   // and candidate cost bits
    int xs[kSmallSet];        // epsilon records (both ends in this set)
    int xd[kSmallSet];
    uint32_t xp[kSmallSet];
};
static_assert(kRing * sizeof(SmallSlot) <= 2 * kLatLds * sizeof(float), "the ring fits the cost half of the LDS");

// Polls of one flag before a pass gives up.
__device__ __forceinline__ long long lat_spin(const Params &p) { return p.lat_spin > 0 ? p.lat_spin : kSmallSpin; }

// Wait until *f >= v (every lane reads the same LDS word); false if the pass
// has failed or the wait gave up (then it marks the pass failed).
__device__ __forceinline__ bool small_wait(int *f, int v, int *fail, long long spin)
{
    for (long long i = 0;; i++) {
        if (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= v) break;
        if (__hip_atomic_load(fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) || i >= spin) {
            __hip_atomic_store(fail, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    return true;
}

// Every record's extra cost from its destination's (stored in e_key by the
// pass that computed the nodes') and the kept arcs of each set, the sets in
// parallel, one wave each: the block pass's arithmetic.
__device__ void lattice_records(const Params &p, const UttLayout &ly, int Tp)
{
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    const float lb = p.lattice_beam;
    const uint32_t *eg = p.e_key + ly.sv0;
    const uint32_t *tok = p.sv_key + ly.sv0;
    unsigned long long *kcnt = reinterpret_cast<unsigned long long *>(p.lo_off + ly.fo0);
    for (int n = wid; n <= Tp; n += nw) {
        const int j = Tp - n;
        const int ne = j < Tp ? static_cast<int>(p.le_cnt[ly.fo0 + j]) : 0;
        const int nx = static_cast<int>(p.lx_cnt[ly.fo0 + j]);
        int kept = 0;
        const int64_t e0 = ly.le0 + (j < Tp ? p.le_off[ly.fo0 + j] : 0);
        for (int i = lane; i < ne; i += kWave) {
            const int4 x = p.lat_e[e0 + i];
            const float d1 = __int_as_float(x.w) - okey_val(tok[x.y]);
            const float ex = d1 + okey_val(ld_relaxed(eg + x.y));
            p.ex_e[e0 + i] = ex;
            kept += ex <= lb;
        }
        const int64_t x0 = ly.lx0 + p.lx_off[ly.fo0 + j];
        for (int i = lane; i < nx; i += kWave) {
            const int4 x = p.lat_x[x0 + i];
            const float d1 = __int_as_float(x.w) - okey_val(tok[x.y]);
            const float ex = d1 + okey_val(ld_relaxed(eg + x.y));
            p.ex_x[x0 + i] = ex;
            kept += ex <= lb;
        }
        const int k = __builtin_amdgcn_readlane(wave_incl_scan(kept), kWave - 1);
        if (lane == 0) kcnt[j] = static_cast<unsigned long long>(k);
    }
    vm_wait();
}

// Called by the whole block when every set holds at most kSmallSet
// survivors, emitting records and epsilon records.
__device__ void lattice_small(const Params &p, int u, uint32_t *s_e, float *s_c)
{
    const long long spin = lat_spin(p);
    UttState &st = p.st[u];
    const UttLayout ly = p.lay[u];
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wid = tid / kWave;
    const int nw = blockDim.x / kWave;
    const int Tp = st.Tp;
    const int64_t *so = p.sv_off + ly.fo0;
    const float lb = p.lattice_beam;
    const float B = st.final_cost;
    const bool use_final = p.g.final_w != nullptr && st.reached_final;
    uint32_t *eg = p.e_key + ly.sv0;
    const uint32_t *tok = p.sv_key + ly.sv0;
    unsigned long long *kcnt = reinterpret_cast<unsigned long long *>(p.lo_off + ly.fo0);
    const uint32_t kinf = okey(__int_as_float(0x7F800000));
    // LDS: extra-cost keys and costs of two sets, the flags, the ring
    uint32_t *se = s_e;
    float *sc = reinterpret_cast<float *>(s_e + 2 * kSmallSet);
    int *filled = reinterpret_cast<int *>(s_e + 4 * kSmallSet);   // per slot: 1 + the last set placed
    int *done = filled + kRing;                                     // sets wave 0 has finished
    int *fail = done + 1;
    SmallSlot *ring = reinterpret_cast<SmallSlot *>(s_c);
    if (tid < kRing) filled[tid] = 0;
    if (tid == 0) {
        *done = 0;
        *fail = 0;
    }
    __syncthreads();

    if (wid > 0) {
        // ---- the loading waves: set n (the n-th from the last) into slot n mod kRing ----
        for (int n = wid - 1; n <= Tp; n += nw - 1) {
            const int slot = n % kRing;
            if (n >= kRing && !small_wait(done, n - kRing + 1, fail, spin)) break;
            const int j = Tp - n;
            const int b0 = static_cast<int>(so[j]);
            const int nB = static_cast<int>(so[j + 1] - so[j]);
            const int ne = j < Tp ? static_cast<int>(p.le_cnt[ly.fo0 + j]) : 0;
            const int nx = static_cast<int>(p.lx_cnt[ly.fo0 + j]);
            uint32_t key = 0;
            int4 e = make_int4(0, 0, 0, 0), x = make_int4(0, 0, 0, 0);
            if (lane < nB) key = tok[b0 + lane];
            if (lane < ne) e = p.lat_e[ly.le0 + p.le_off[ly.fo0 + j] + lane];
            if (lane < nx) x = p.lat_x[ly.lx0 + p.lx_off[ly.fo0 + j] + lane];
            SmallSlot &sl = ring[slot];
            sl.key[lane] = key;
            sl.es[lane] = e.x;
            sl.ed[lane] = e.y;
            sl.ep[lane] = static_cast<uint32_t>(e.w);
            sl.xs[lane] = x.x;
            sl.xd[lane] = x.y;
            sl.xp[lane] = static_cast<uint32_t>(x.w);
            if (lane == 0) {
                sl.b0 = b0;
                sl.nB = nB;
                sl.ne = ne;
                sl.nx = nx;
            }
            // the slot's contents before its flag
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            if (lane == 0) __hip_atomic_store(filled + slot, n + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
    } else {
        // ---- wave 0: the sets from last to first (the block pass's steps) ----
        int hA = 0, a0 = 0;   // the half holding S_j+1, and its first survivor
        for (int n = 0; n <= Tp; n++) {
            const int j = Tp - n;
            const SmallSlot &sl = ring[n % kRing];
            if (!small_wait(filled + n % kRing, n + 1, fail, spin)) break;
            const int b0 = sl.b0, nB = sl.nB, ne = sl.ne, nx = sl.nx;
            const int hB = hA ^ 1;
            uint32_t *eA = se + hA * kSmallSet, *eB = se + hB * kSmallSet;
            float *cA = sc + hA * kSmallSet, *cB = sc + hB * kSmallSet;
            if (lane < nB) {
                const float c = okey_val(sl.key[lane]);
                cB[lane] = c;
                uint32_t e0 = kinf;
                if (j == Tp) {
                    const float f = use_final ? p.g.final_w[p.sv_state[ly.sv0 + b0 + lane]] : 0.0f;
                    e0 = okey((c + f) - B);
                }
                eB[lane] = e0;
            }
            wave_lds_handover();
            // emitting arcs into S_j+1
            if (lane < ne) {
                const int d = sl.ed[lane] - a0;
                const float d1 = __uint_as_float(sl.ep[lane]) - cA[d];
                const float ex = d1 + okey_val(eA[d]);
                atomicMin(eB + (sl.es[lane] - b0), okey(ex));
            }
            wave_lds_handover();
            // epsilon arcs inside S_j, to their fixed point
            while (nx > 0) {
                bool changed = false;
                if (lane < nx) {
                    const int d = sl.xd[lane] - b0;
                    const float d1 = __uint_as_float(sl.xp[lane]) - cB[d];
                    const float ex = d1 + okey_val(eB[d]);
                    const uint32_t k = okey(ex);
                    if (k < eB[sl.xs[lane] - b0]) {
                        atomicMin(eB + (sl.xs[lane] - b0), k);
                        changed = true;
                    }
                }
                wave_lds_handover();
                if (!__ballot(changed)) break;
            }
            // S_j's extra costs, for the records below
            if (lane < nB) eg[b0 + lane] = eB[lane];
            // the slot has been read: it may take a later set
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            if (lane == 0) __hip_atomic_store(done, n + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            hA = hB;
            a0 = b0;
        }
    }
    // every node's extra cost is stored before any record reads it
    block_sync_vm();
    if (*fail) {
        if (tid == 0) set_status(st, kStatusLatticeWait);
        return;
    }
    lattice_records(p, ly, Tp);
}

// ---------------------------------------------------------------------------
// The backward pass of an utterance with larger sets: at most kLatLds
// survivors and ring-capacity epsilon records each.  The roles are the
// one-wave pass's, with a stream in place of fixed slots.  A set's stream
// holds, in this order, the initial extra-cost keys of its survivors (the
// last set only), its emitting records and its epsilon records, each an
// 8-byte entry: the source's and destination's offsets in their sets and the
// record's first difference fl(p - c(d)), which the loading waves compute
// from device memory.  Every set's place in the stream is the prefix of the
// sizes before it, computed up front, so the loading waves (wave w of W takes
// the sets w-1, w-1+(W-1), ...) write side by side into a ring of LDS entries, 512
// at a time, each piece once wave 0 has read what those ring positions held
// before.  Wave 0 takes the sets in order and the pieces as they arrive; it
// computes the nodes' extra costs as the block pass does and, on the way,
// every record's extra cost (an epsilon record's from the round that changed
// nothing) and the kept arcs of the set, so the records are read once.  The
// arithmetic is the block pass's, step for step.  Every wait is bounded.
//
// Progress: wave 0 waits only for the loader of its current set, which has
// finished its earlier sets (wave 0 has read them) and waits, if at all, for
// ring positions at most a piece ahead of wave 0's, or, for the epsilon
// records (read until the set is done), at most the ring's capacity ahead.
// ---------------------------------------------------------------------------
constexpr int kPipeCap = 8192;     // ring entries (8 bytes each): the cost half of the LDS
constexpr int kPipePiece = 512;    // entries per hand-over (8 per lane)
constexpr int kPipeSlots = 32;     // sets described ahead of wave 0
constexpr int kPipeAvg = 480;      // stream entries per set up to which the pass beats the block pass
static_assert(kPipeCap * sizeof(uint2) == 2 * kLatLds * sizeof(float), "the ring is the cost half of the LDS");
static_assert(kLatLds <= 65536, "a survivor's offset in its set fits 16 bits");

struct PipeMeta {
    int64_t re, rx;       // the set's first emitting and first epsilon record
    int b0, nB, ne, nx;   // first survivor (utterance-relative) and the counts
    int start;            // the set's first stream position
    int pad;
};

// The lattice block's LDS control words.
struct LatCtl {
    PipeMeta meta[kPipeSlots];
    int filled[kPipeSlots];   // per slot: 1 + the last set described there
    int prog[kPipeSlots];     // per slot: stream position up to which its set is written
    int done;                 // sets wave 0 has finished
    int consumed;             // stream position up to which wave 0 has read
    int fail;
    int mB, mE, mX;           // largest set, emitting and epsilon record counts
    unsigned long long total; // stream entries of the utterance
};

// Wait until *f >= v; LDS-only ordering (the waiting wave's device-memory
// stores are not waited for).  False if the pass has failed or the wait gave
// up (then it marks the pass failed).
__device__ __forceinline__ bool pipe_wait(const int *f, int v, int *fail, long long spin)
{
    for (long long i = 0;; i++) {
        if (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= v) break;
        if (__hip_atomic_load(fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) || i >= spin) {
            __hip_atomic_store(fail, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    return true;
}

// The wave's LDS accesses so far, then *f = v.
__device__ __forceinline__ void pipe_publish(int *f, int v)
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    if (lane_id() == 0) __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// A loading wave: sets pw, pw + np, ... into the stream.
__device__ void pipe_load(const Params &p, const UttLayout &ly, const UttState &st, LatCtl *ctl, uint2 *ring,
                          int pw, int np)
{
    const long long spin = lat_spin(p);
    const int lane = lane_id();
    const int Tp = st.Tp;
    const float B = st.final_cost;
    const bool use_final = p.g.final_w != nullptr && st.reached_final;
    const int64_t *so = p.sv_off + ly.fo0;
    const uint32_t *tok = p.sv_key + ly.sv0;
    const unsigned long long *start_of = reinterpret_cast<const unsigned long long *>(p.lo_off + ly.fo0);
    constexpr int kQ = kPipePiece / kWave;
    for (int n = pw; n <= Tp; n += np) {
        const int j = Tp - n;
        const int slot = n % kPipeSlots;
        const int b0 = static_cast<int>(so[j]);
        const int b1 = static_cast<int>(so[j + 1]);
        const int nB = b1 - b0;
        const int ne = j < Tp ? static_cast<int>(p.le_cnt[ly.fo0 + j]) : 0;
        const int nx = static_cast<int>(p.lx_cnt[ly.fo0 + j]);
        const int64_t re = ly.le0 + (j < Tp ? p.le_off[ly.fo0 + j] : 0);
        const int64_t rx = ly.lx0 + p.lx_off[ly.fo0 + j];
        const int start = static_cast<int>(ld_relaxed(start_of + j));
        if (n >= kPipeSlots && !pipe_wait(&ctl->done, n - kPipeSlots + 1, &ctl->fail, spin)) return;
        if (lane == 0) {
            PipeMeta &m = ctl->meta[slot];
            m.re = re;
            m.rx = rx;
            m.b0 = b0;
            m.nB = nB;
            m.ne = ne;
            m.nx = nx;
            m.start = start;
            ctl->prog[slot] = start;
        }
        pipe_publish(ctl->filled + slot, n + 1);
        int pos = start;
        if (n == 0) {
            // the last set: fl(fl(c + f) - B) of every survivor
            for (int i0 = 0; i0 < nB; i0 += kPipePiece) {
                uint32_t v[kQ];
#pragma unroll
                for (int q = 0; q < kQ; q++) {
                    const int i = i0 + q * kWave + lane;
                    v[q] = 0;
                    if (i < nB) {
                        const float c = okey_val(tok[b0 + i]);
                        const float f = use_final ? p.g.final_w[p.sv_state[ly.sv0 + b0 + i]] : 0.0f;
                        v[q] = okey((c + f) - B);
                    }
                }
                const int end = start + min(i0 + kPipePiece, nB);
                if (!pipe_wait(&ctl->consumed, end - kPipeCap, &ctl->fail, spin)) return;
#pragma unroll
                for (int q = 0; q < kQ; q++) {
                    const int i = i0 + q * kWave + lane;
                    if (i < nB) ring[(start + i) & (kPipeCap - 1)] = make_uint2(v[q], 0u);
                }
                pipe_publish(ctl->prog + slot, end);
            }
            pos += nB;
        }
        // the records: emitting (destination in S_j+1), then epsilon
        const int nr = ne + nx;
        for (int i0 = 0; i0 < nr; i0 += kPipePiece) {
            int4 x[kQ];
#pragma unroll
            for (int q = 0; q < kQ; q++) {
                const int i = i0 + q * kWave + lane;
                x[q] = make_int4(0, 0, 0, 0);
                if (i < ne) x[q] = p.lat_e[re + i];
                else if (i < nr) x[q] = p.lat_x[rx + (i - ne)];
            }
            uint2 v[kQ];
#pragma unroll
            for (int q = 0; q < kQ; q++) {
                const int i = i0 + q * kWave + lane;
                v[q] = make_uint2(0u, 0u);
                if (i < nr) {
                    const float d1 = __int_as_float(x[q].w) - okey_val(tok[x[q].y]);
                    const int base = i < ne ? b1 : b0;
                    v[q] = make_uint2(static_cast<uint32_t>(x[q].x - b0) << 16 | static_cast<uint32_t>(x[q].y - base),
                                      __float_as_uint(d1));
                }
            }
            const int end = pos + min(i0 + kPipePiece, nr);
            if (!pipe_wait(&ctl->consumed, end - kPipeCap, &ctl->fail, spin)) return;
#pragma unroll
            for (int q = 0; q < kQ; q++) {
                const int i = i0 + q * kWave + lane;
                if (i < nr) ring[(pos + i) & (kPipeCap - 1)] = v[q];
            }
            pipe_publish(ctl->prog + slot, end);
        }
    }
}

// Wave 0's wait for stream position `end` of the set in `slot`: `have` is
// the position it last saw written.  Before it blocks it reports what it has
// read (up to `cur`), which the loaders may be waiting for.
__device__ __forceinline__ bool pipe_need(LatCtl *ctl, int slot, int end, int &have, int cur, long long spin)
{
    if (have >= end) return true;
    pipe_publish(&ctl->consumed, cur);
    for (long long i = 0;; i++) {
        const int v = __hip_atomic_load(ctl->prog + slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (v >= end) {
            have = v;
            break;
        }
        if (__hip_atomic_load(&ctl->fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) || i >= spin) {
            __hip_atomic_store(&ctl->fail, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    return true;
}

// kQ entries per lane of a set's emitting records for wave 0: entries i0..
// of the region starting at stream position r; kFull when all of them exist,
// else the missing lanes repeat the region's last entry with a key that
// lowers nothing.  The loads carry no condition, so they are issued together.
template <bool kFull, int kQ>
__device__ __forceinline__ void pipe_emit(const uint2 *ring, int r, int i0, int ne, const uint32_t *eA, uint32_t *eB,
                                          float *exo, float lb, int &kept)
{
    const int lane = lane_id();
    uint2 v[kQ];
#pragma unroll
    for (int q = 0; q < kQ; q++) {
        const int i = i0 + q * kWave + lane;
        v[q] = ring[(r + (kFull ? i : min(i, ne - 1))) & (kPipeCap - 1)];
    }
    float ex[kQ];
#pragma unroll
    for (int q = 0; q < kQ; q++) ex[q] = __uint_as_float(v[q].y) + okey_val(eA[v[q].x & 0xFFFFu]);
#pragma unroll
    for (int q = 0; q < kQ; q++) {
        const int i = i0 + q * kWave + lane;
        const bool ok = kFull || i < ne;
        atomicMin(eB + (v[q].x >> 16), ok ? okey(ex[q]) : 0xFFFFFFFFu);
        if (ok) exo[i] = ex[q];
        kept += ok && ex[q] <= lb;
    }
}

// The same for an epsilon round.
template <bool kFull, int kQ>
__device__ __forceinline__ void pipe_eps(const uint2 *ring, int r, int i0, int nx, uint32_t *eB, float *exo, float lb,
                                         int &kx, bool &changed)
{
    const int lane = lane_id();
    uint2 v[kQ];
#pragma unroll
    for (int q = 0; q < kQ; q++) {
        const int i = i0 + q * kWave + lane;
        v[q] = ring[(r + (kFull ? i : min(i, nx - 1))) & (kPipeCap - 1)];
    }
    uint32_t ed[kQ], es[kQ];
#pragma unroll
    for (int q = 0; q < kQ; q++) {
        ed[q] = eB[v[q].x & 0xFFFFu];
        es[q] = eB[v[q].x >> 16];
    }
#pragma unroll
    for (int q = 0; q < kQ; q++) {
        const int i = i0 + q * kWave + lane;
        const bool ok = kFull || i < nx;
        const float ex = __uint_as_float(v[q].y) + okey_val(ed[q]);
        const uint32_t k = okey(ex);
        if (ok && k < es[q]) {
            atomicMin(eB + (v[q].x >> 16), k);
            changed = true;
        }
        if (ok) exo[i] = ex;
        kx += ok && ex <= lb;
    }
}

__device__ __forceinline__ int64_t uniform64(int64_t v)
{
    const uint64_t u = static_cast<uint64_t>(v);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Wave 0: the sets from last to first.
__device__ void pipe_chain(const Params &p, const UttLayout &ly, int Tp, LatCtl *ctl, const uint2 *ring,
                           uint32_t *se)
{
    const long long spin = lat_spin(p);
    const int lane = lane_id();
    const float lb = p.lattice_beam;
    const uint32_t kinf = okey(__int_as_float(0x7F800000));
    unsigned long long *kcnt = reinterpret_cast<unsigned long long *>(p.lo_off + ly.fo0);
    constexpr int kQ = kPipePiece / kWave;
    int hA = 0;   // the half holding S_j+1
    for (int n = 0; n <= Tp; n++) {
        const int j = Tp - n;
        const int slot = n % kPipeSlots;
        if (!pipe_wait(ctl->filled + slot, n + 1, &ctl->fail, spin)) return;
        const PipeMeta &mm = ctl->meta[slot];
        const int nB = __builtin_amdgcn_readfirstlane(mm.nB);
        const int ne = __builtin_amdgcn_readfirstlane(mm.ne);
        const int nx = __builtin_amdgcn_readfirstlane(mm.nx);
        const int start = __builtin_amdgcn_readfirstlane(mm.start);
        float *exe = p.ex_e + uniform64(mm.re);
        float *exx = p.ex_x + uniform64(mm.rx);
        const int hB = hA ^ 1;
        const uint32_t *eA = se + hA * kLatLds;
        uint32_t *eB = se + hB * kLatLds;
        int pos = start;
        int have = start;
        if (n == 0) {
            for (int i0 = 0; i0 < nB; i0 += kPipePiece) {
                if (!pipe_need(ctl, slot, pos + min(i0 + kPipePiece, nB), have, pos + i0, spin)) return;
                uint32_t v[kQ];
#pragma unroll
                for (int q = 0; q < kQ; q++) v[q] = ring[(pos + min(i0 + q * kWave + lane, nB - 1)) & (kPipeCap - 1)].x;
#pragma unroll
                for (int q = 0; q < kQ; q++) eB[min(i0 + q * kWave + lane, nB - 1)] = v[q];
            }
            pos += nB;
        } else {
            for (int i0 = 0; i0 < nB; i0 += 2 * kWave) {
                eB[min(i0 + lane, nB - 1)] = kinf;
                eB[min(i0 + kWave + lane, nB - 1)] = kinf;
            }
        }
        wave_lds_handover();
        int kept = 0;
        // emitting arcs into S_j+1
        for (int i0 = 0; i0 < ne; i0 += kPipePiece) {
            const int left = ne - i0;
            if (!pipe_need(ctl, slot, pos + min(i0 + kPipePiece, ne), have, pos + i0, spin)) return;
            if (left >= kPipePiece) pipe_emit<true, kQ>(ring, pos, i0, ne, eA, eB, exe, lb, kept);
            else if (left > 4 * kWave) pipe_emit<false, kQ>(ring, pos, i0, ne, eA, eB, exe, lb, kept);
            else if (left > 2 * kWave) pipe_emit<false, 4>(ring, pos, i0, ne, eA, eB, exe, lb, kept);
            else if (left > kWave) pipe_emit<false, 2>(ring, pos, i0, ne, eA, eB, exe, lb, kept);
            else pipe_emit<false, 1>(ring, pos, i0, ne, eA, eB, exe, lb, kept);
            // what has been read may be refilled (not after the last piece:
            // the set's end reports it)
            if (left > kPipePiece) pipe_publish(&ctl->consumed, pos + i0 + kPipePiece);
        }
        pos += ne;
        wave_lds_handover();
        // epsilon arcs inside S_j, to their fixed point; the round that
        // changes nothing stores the final extra costs last
        if (nx > 0) {
            if (!pipe_need(ctl, slot, pos + nx, have, pos, spin)) return;
            int kx = 0;
            for (;;) {
                bool changed = false;
                kx = 0;
                for (int i0 = 0; i0 < nx; i0 += kPipePiece) {
                    const int left = nx - i0;
                    if (left >= kPipePiece) pipe_eps<true, kQ>(ring, pos, i0, nx, eB, exx, lb, kx, changed);
                    else if (left > 4 * kWave) pipe_eps<false, kQ>(ring, pos, i0, nx, eB, exx, lb, kx, changed);
                    else if (left > 2 * kWave) pipe_eps<false, 4>(ring, pos, i0, nx, eB, exx, lb, kx, changed);
                    else if (left > kWave) pipe_eps<false, 2>(ring, pos, i0, nx, eB, exx, lb, kx, changed);
                    else pipe_eps<false, 1>(ring, pos, i0, nx, eB, exx, lb, kx, changed);
                }
                wave_lds_handover();
                if (!__ballot(changed)) break;
            }
            kept += kx;
            pos += nx;
        }
        const int k = __builtin_amdgcn_readlane(wave_incl_scan(kept), kWave - 1);
        if (lane == 0) kcnt[j] = static_cast<unsigned long long>(k);
        // the set's entries are read: the loaders may reuse them and its slot
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        if (lane == 0) {
            __hip_atomic_store(&ctl->consumed, pos, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            __hip_atomic_store(&ctl->done, n + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        hA = hB;
    }
}

// Called by the whole block when the pass applies (see the caller).
__device__ void lattice_pipe(const Params &p, int u, uint32_t *s_e, float *s_c, int *sh, LatCtl *ctl)
{
    UttState &st = p.st[u];
    const UttLayout ly = p.lay[u];
    const int tid = threadIdx.x;
    const int wid = tid / kWave;
    const int nw = blockDim.x / kWave;
    const int Tp = st.Tp;
    const int64_t *so = p.sv_off + ly.fo0;
    unsigned long long *start_of = reinterpret_cast<unsigned long long *>(p.lo_off + ly.fo0);
    // every set's first stream position (in the kept-count words, which the
    // pass overwrites once the set is done)
    int carry = 0;
    for (int n0 = 0; n0 <= Tp; n0 += blockDim.x) {
        const int n = n0 + tid;
        int sz = 0;
        if (n <= Tp) {
            const int j = Tp - n;
            sz = static_cast<int>((n == 0 ? so[j + 1] - so[j] : 0) + (j < Tp ? p.le_cnt[ly.fo0 + j] : 0) +
                                  p.lx_cnt[ly.fo0 + j]);
        }
        int total;
        const int ex = block_excl_scan(sz, sh + 4, &total);
        if (n <= Tp) start_of[Tp - n] = static_cast<unsigned long long>(carry + ex);
        carry += total;
    }
    if (tid < kPipeSlots) {
        ctl->filled[tid] = 0;
        ctl->prog[tid] = 0;
    }
    if (tid == 0) {
        ctl->done = 0;
        ctl->consumed = 0;
        ctl->fail = 0;
    }
    block_sync_vm();
    uint2 *ring = reinterpret_cast<uint2 *>(s_c);
    if (wid == 0) pipe_chain(p, ly, Tp, ctl, ring, s_e);
    else pipe_load(p, ly, st, ctl, ring, wid - 1, nw - 1);
    vm_wait();
    __syncthreads();
    if (ctl->fail && tid == 0) set_status(st, kStatusLatticeWait);
}

// Lattice-beam pruning of utterance u by one block: the one-wave pass when
// every set is small, else the streamed pass when every set fits it, else the
// block pass; then the kept counts become the output offsets.
__device__ void lattice_block(const Params &p, int u, uint32_t *s_e, float *s_c, int *sh, LatCtl *ctl)
{
    UttState &st = p.st[u];
    const UttLayout ly = p.lay[u];
    const int tid = threadIdx.x;
    const int nw = blockDim.x / kWave;
    const int Tp = st.Tp;
    const int64_t *so = p.sv_off + ly.fo0;
    unsigned long long *kcnt = reinterpret_cast<unsigned long long *>(p.lo_off + ly.fo0);
    // the largest set and record counts, and the streamed pass's total
    if (tid == 0) {
        ctl->mB = ctl->mE = ctl->mX = 0;
        ctl->total = 0;
    }
    __syncthreads();
    {
        int64_t mb = 0, me = 0, mx = 0;
        unsigned long long tot = 0;
        for (int j = tid; j <= Tp; j += blockDim.x) {
            const int64_t nB = so[j + 1] - so[j];
            const int64_t ne = j < Tp ? p.le_cnt[ly.fo0 + j] : 0;
            const int64_t nx = p.lx_cnt[ly.fo0 + j];
            mb = max(mb, nB);
            me = max(me, ne);
            mx = max(mx, nx);
            tot += static_cast<unsigned long long>((j == Tp ? nB : 0) + ne + nx);
        }
        constexpr int64_t kBig = 1 << 30;
        atomicMax(&ctl->mB, static_cast<int>(min(mb, kBig)));
        atomicMax(&ctl->mE, static_cast<int>(min(me, kBig)));
        atomicMax(&ctl->mX, static_cast<int>(min(mx, kBig)));
        atomicAdd(&ctl->total, tot);
    }
    __syncthreads();
    const int mB = ctl->mB, mE = ctl->mE, mX = ctl->mX;
    const bool small = nw > 1 && p.lat_lds >= kSmallSet && mB <= kSmallSet && mE <= kSmallSet && mX <= kSmallSet;
    // The streamed pass's time grows with the records, the block pass's
    // mostly with the sets: the streamed one where sets are small on average
    // (or wherever it fits when lat_pipe > 0).
    const unsigned long long tot = ctl->total;
    const bool piped = nw > 1 && p.lat_pipe >= 0 && mB <= min(kLatLds, p.lat_lds) && mX <= kPipeCap &&
                       tot < (1ull << 30) &&
                       (p.lat_pipe > 0 || tot <= static_cast<unsigned long long>(kPipeAvg) * (Tp + 1));
    if (small) lattice_small(p, u, s_e, s_c);
    else if (piped) lattice_pipe(p, u, s_e, s_c, sh, ctl);
    else lattice_sets(p, u, s_e, s_c, sh);
    __syncthreads();
    // kept arcs per set -> output offsets (exclusive prefix over the sets)
    int64_t carry = 0;
    for (int j0 = 0; j0 <= Tp; j0 += blockDim.x) {
        const int j = j0 + tid;
        const int64_t c = j <= Tp ? static_cast<int64_t>(ld_relaxed(kcnt + j)) : 0;
        int total;
        const int ex = block_excl_scan(static_cast<int>(c), sh + 4, &total);
        if (j <= Tp) p.lo_off[ly.fo0 + j] = carry + ex;
        carry += total;
    }
    if (tid == 0) {
        p.lo_off[ly.fo0 + Tp + 1] = carry;
        st.lat_kept = carry;
    }
}

// Blocks [0, U): backtrace of utterance b; blocks [U, 2U) (with a lattice):
// lattice-beam pruning of utterance b - U.  The two are independent and run
// side by side.
__global__ __launch_bounds__(kLatT) void finish_kernel(Params p)
{
    __shared__ __align__(16) uint32_t s_e[2 * kLatLds];
    __shared__ __align__(16) float s_c[2 * kLatLds];
    __shared__ __align__(8) int sh[24];   // flags, a 64-bit count, scan scratch (17 ints)
    __shared__ LatCtl ctl;
    const int b = blockIdx.x;
    const int u = b < p.U ? b : b - p.U;
    if (p.st[u].status != 0) return;
    if (threadIdx.x == 0) {
        sh[0] = 0;
        *reinterpret_cast<long long *>(sh + 2) = 0;
    }
    __syncthreads();
    const uint64_t t0 = p.profile ? wall_clock64() : 0;
    if (b < p.U) backtrace_block(p, u, sh);
    else lattice_block(p, u, s_e, s_c, sh, &ctl);
    if (p.profile && threadIdx.x == 0) p.st[u].finish_ticks[b < p.U ? 0 : 1] = wall_clock64() - t0;
}

__device__ __forceinline__ void cas16(int4 *v, int i, int j)
{
    int4 a = v[i], b = v[j];
    if (b.y < a.y) {
        v[i] = b;
        v[j] = a;
    }
}

// Ascending sort of n records by arc id (unique within a token set) by the
// whole block: the bitonic network in its "flip" form, where every
// comparator puts the smaller key first, so positions >= n act as +inf and
// are never touched.
__device__ void sort_records(int4 *v, int n)
{
    int n2 = 1;
    while (n2 < n) n2 <<= 1;
    for (int size = 2; size <= n2; size <<= 1) {
        const int half = size >> 1;
        for (int t = threadIdx.x; t < n2 / 2; t += blockDim.x) {
            int i = (t / half) * size + (t % half);
            int j = (t / half) * size + size - 1 - (t % half);
            if (j < n) cas16(v, i, j);
        }
        __syncthreads();
        for (int d = half >> 1; d >= 1; d >>= 1) {
            for (int t = threadIdx.x; t < n2 / 2; t += blockDim.x) {
                int i = (t / d) * 2 * d + (t % d);
                int j = i + d;
                if (j < n) cas16(v, i, j);
            }
            __syncthreads();
        }
    }
}

constexpr int kEmitK = 512;     // kept arcs of a set that one wave sorts in LDS
constexpr int kEmitW = 4;       // waves per block of the output pass
constexpr int kEmitQ = 4;       // records per lane in flight in the scan
constexpr int kEmitDefer = 256; // larger sets a block keeps for its joint pass

// A set's record offsets, loaded a set ahead of their use.
struct EmitMeta {
    int64_t o0, o1;   // output range (kept-arc offsets)
    int64_t e0, x0;   // first emitting and first epsilon record
    int64_t ne, nx;
};

__device__ __forceinline__ EmitMeta emit_meta(const Params &p, const UttLayout &ly, int j, int Tp)
{
    EmitMeta m;
    m.o0 = p.lo_off[ly.fo0 + j];
    m.o1 = p.lo_off[ly.fo0 + j + 1];
    m.e0 = ly.le0 + (j < Tp ? p.le_off[ly.fo0 + j] : 0);
    m.ne = j < Tp ? p.le_cnt[ly.fo0 + j] : 0;
    m.x0 = ly.lx0 + p.lx_off[ly.fo0 + j];
    m.nx = p.lx_cnt[ly.fo0 + j];
    return m;
}

// A set with more kept arcs than a wave's buffer, by one wave: each kept
// record's rank is the number of kept records of smaller arc (only when the
// block's list of such sets is full).
__device__ void emit_set_counted(const Params &p, const EmitMeta &c, int j, int n, int4 *out)
{
    const int lane = lane_id();
    const float lb = p.lattice_beam;
    const int ne = static_cast<int>(c.ne);
    const int nr = ne + static_cast<int>(c.nx);
    for (int a0 = 0; a0 < nr; a0 += kWave) {
        const int a = a0 + lane;
        bool ka = false;
        float xa = 0.0f;
        int4 ra = make_int4(0, 0, 0, 0);
        if (a < nr) {
            xa = a < ne ? p.ex_e[c.e0 + a] : p.ex_x[c.x0 + (a - ne)];
            ka = xa <= lb;
            if (ka) ra = a < ne ? p.lat_e[c.e0 + a] : p.lat_x[c.x0 + (a - ne)];
        }
        if (!__ballot(ka)) continue;
        int rank = 0;
        for (int b0 = 0; b0 < nr; b0 += kWave) {
            const int b = b0 + lane;
            int arc = 0x7FFFFFFF;   // not kept: larger than every arc
            if (b < nr) {
                const float xb = b < ne ? p.ex_e[c.e0 + b] : p.ex_x[c.x0 + (b - ne)];
                if (xb <= lb) arc = (b < ne ? p.lat_e[c.e0 + b] : p.lat_x[c.x0 + (b - ne)]).z;
            }
            for (int l = 0; l < kWave; l++) rank += __builtin_amdgcn_readlane(arc, l) < ra.z;
        }
        if (ka && rank < n) out[rank] = make_int4(j, ra.z, ra.w, __float_as_int(xa));
    }
}

// The sorted lattice output: {frame, arc, cost, extra} of every kept arc,
// each set's arcs in ascending arc order (arc ids are unique within a set).
// A wave takes every (gridDim.x * kEmitW)-th set of its utterance: it scans
// the set's extra costs, places the kept records in its LDS buffer by their
// order in the scan, and writes each to its rank among them.  Sets with more
// kept arcs than a wave's buffer wait in a list for the whole block, which
// then gathers each into the four buffers together (or, beyond those, into
// the output itself) and sorts it with the bitonic network.
__global__ __launch_bounds__(kEmitW * kWave) void lattice_emit_kernel(Params p)
{
    __shared__ int4 buf[kEmitW * kEmitK];
    __shared__ int defer[kEmitDefer];
    __shared__ int n_defer, sh_n;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int u = blockIdx.y;
    const UttState &st = p.st[u];
    if (st.status != 0) return;
    const UttLayout &ly = p.lay[u];
    const int Tp = st.Tp;
    const float lb = p.lattice_beam;
    const int step = gridDim.x * kEmitW;
    if (threadIdx.x == 0) n_defer = 0;
    __syncthreads();
    int4 *wb = buf + w * kEmitK;
    int j = blockIdx.x * kEmitW + w;
    EmitMeta m{};
    if (j <= Tp) m = emit_meta(p, ly, j, Tp);
    for (; j <= Tp; j += step) {
        const EmitMeta c = m;
        if (j + step <= Tp) m = emit_meta(p, ly, j + step, Tp);
        const int n = static_cast<int>(c.o1 - c.o0);
        int4 *out = p.lat_out + ly.lo0 + c.o0;
        const int ne = static_cast<int>(c.ne);
        const int nr = ne + static_cast<int>(c.nx);
        if (n <= 0 || nr <= 0) continue;
        if (n > kEmitK) {
            int d = 0;
            if (lane == 0) d = atomicAdd(&n_defer, 1);
            d = __builtin_amdgcn_readfirstlane(d);
            if (d < kEmitDefer) {
                if (lane == 0) defer[d] = j;
            } else {
                emit_set_counted(p, c, j, n, out);
            }
            continue;
        }
        int cnt = 0;
        for (int i0 = 0; i0 < nr; i0 += kEmitQ * kWave) {
            float x[kEmitQ];
#pragma unroll
            for (int q = 0; q < kEmitQ; q++) {
                const int i = min(i0 + q * kWave + lane, nr - 1);
                x[q] = i < ne ? p.ex_e[c.e0 + i] : p.ex_x[c.x0 + (i - ne)];
            }
#pragma unroll
            for (int q = 0; q < kEmitQ; q++) {
                const int i = i0 + q * kWave + lane;
                const bool kp = i < nr && x[q] <= lb;
                const uint64_t km = __ballot(kp);
                const int slot = cnt + __popcll(km & lanemask_lt());
                if (kp && slot < kEmitK) {
                    const int4 r = i < ne ? p.lat_e[c.e0 + i] : p.lat_x[c.x0 + (i - ne)];
                    wb[slot] = make_int4(j, r.z, r.w, __float_as_int(x[q]));
                }
                cnt += __popcll(km);
            }
        }
        wave_lds_handover();
        const int m2 = min(cnt, n);
        for (int a = lane; a < m2; a += kWave) {
            const int4 e = wb[a];
            int rank = 0;
            for (int b = 0; b < m2; b++) rank += wb[b].y < e.y;
            out[rank] = e;
        }
        wave_lds_handover();
    }
    // the block's large sets, one after another
    __syncthreads();
    const int nd = min(n_defer, kEmitDefer);
    for (int d = 0; d < nd; d++) {
        const int jd = defer[d];
        const EmitMeta c = emit_meta(p, ly, jd, Tp);
        const int n = static_cast<int>(c.o1 - c.o0);
        int4 *out = p.lat_out + ly.lo0 + c.o0;
        int4 *v = n <= kEmitW * kEmitK ? buf : out;
        if (threadIdx.x == 0) sh_n = 0;
        __syncthreads();
        const int ne = static_cast<int>(c.ne);
        const int nr = ne + static_cast<int>(c.nx);
        for (int i = threadIdx.x; i < nr; i += blockDim.x) {
            const float x = i < ne ? p.ex_e[c.e0 + i] : p.ex_x[c.x0 + (i - ne)];
            if (x <= lb) {
                const int slot = atomicAdd(&sh_n, 1);
                const int4 r = i < ne ? p.lat_e[c.e0 + i] : p.lat_x[c.x0 + (i - ne)];
                if (slot < n) v[slot] = make_int4(jd, r.z, r.w, __float_as_int(x));
            }
        }
        __syncthreads();
        sort_records(v, n);
        if (v == buf)
            for (int i = threadIdx.x; i < n; i += blockDim.x) out[i] = buf[i];
        __syncthreads();
    }
}

// The best paths of all utterances packed one after another (utterance
// order, each path in order), so that the host copies them at once.  One
// block: offsets by a block scan over the utterances, then the block copies
// each path.
__global__ __launch_bounds__(1024) void pack_paths_kernel(Params p)
{
    __shared__ int sh_scan[17];
    __shared__ int64_t sh_off[1024];
    __shared__ int sh_len[1024];
    int64_t carry = 0;
    for (int u0 = 0; u0 < p.U; u0 += blockDim.x) {
        const int u = u0 + threadIdx.x;
        const int len = u < p.U && p.st[u].status == WFST_OK ? p.st[u].path_len : 0;
        int total;
        const int ex = block_excl_scan(len, sh_scan, &total);
        sh_off[threadIdx.x] = carry + ex;
        sh_len[threadIdx.x] = len;
        carry += total;
        __syncthreads();
        const int nu = min(static_cast<int>(blockDim.x), p.U - u0);
        for (int v = 0; v < nu; v++) {
            const UttLayout &ly = p.lay[u0 + v];
            const int lv = sh_len[v];
            const int64_t src = ly.path0 + ly.pathcap - lv;
            for (int i = threadIdx.x; i < lv; i += blockDim.x)
                p.path_packed[sh_off[v] + i] = make_int2(p.path_arc[src + i], p.path_frame[src + i]);
        }
        __syncthreads();
    }
}

// Zero a buffer (a kernel rather than a memset node, so the decode's
// enqueued work is kernels and copies only).
__global__ __launch_bounds__(256) void zero_kernel(uint4 *p, int64_t n16, uint32_t *tail, int ntail)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
    if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < ntail) tail[threadIdx.x] = 0u;
}

}  // namespace

hipError_t launch_zero(void *ptr, size_t bytes, hipStream_t s)
{
    // ptr is 256-byte aligned (arena carving) and bytes a multiple of 4
    if (bytes == 0) return hipSuccess;
    const int64_t n16 = static_cast<int64_t>(bytes / 16);
    const int ntail = static_cast<int>((bytes % 16) / 4);
    uint32_t *tail = reinterpret_cast<uint32_t *>(static_cast<char *>(ptr) + n16 * 16);
    const int64_t blocks = std::min<int64_t>(std::max<int64_t>((n16 + 255) / 256, 1), 1024);
    hipLaunchKernelGGL(zero_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, static_cast<uint4 *>(ptr),
                       n16, tail, ntail);
    return hipGetLastError();
}

hipError_t launch_final(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(final_kernel, dim3(p.U), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_pack_paths(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(pack_paths_kernel, dim3(1), dim3(1024), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_finish(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(finish_kernel, dim3(p.lattice ? 2 * p.U : p.U), dim3(kLatT), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_lattice_emit(const Params &p, int max_frames, hipStream_t s)
{
    // about 1,024 blocks over the batch, no more waves per utterance than sets
    const int sets = max_frames + 1;
    const int g = std::max(1, std::min((1024 + p.U - 1) / p.U, (sets + kEmitW - 1) / kEmitW));
    hipLaunchKernelGGL(lattice_emit_kernel, dim3(g, p.U), dim3(kEmitW * kWave), 0, s, p);
    return hipGetLastError();
}

}  // namespace wfd
