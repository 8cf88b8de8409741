// End-of-utterance kernels: finalTransition and backtrace (Alg. 1 of the
// paper), lattice-beam pruning of the recorded lattice (the backward pass of
// exact lattice generation, Sec. 1 and Sec. 3), and the sorted lattice output.
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
            float c = tok_cost(p.sv_tok[ly.sv0 + i]);
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

// backtrace: follow survivor back-pointers from the final token; arcs are
// written from the end of the utterance's path region backwards.
__global__ void backtrace_kernel(Params p)
{
    const int u = blockIdx.x * blockDim.x + threadIdx.x;
    if (u >= p.U) return;
    UttState &st = p.st[u];
    if (st.status != 0) return;
    const UttLayout &ly = p.lay[u];
    int64_t i = st.final_sv;
    int j = st.Tp;
    int cnt = 0;
    const int64_t end = ly.path0 + ly.pathcap;
    while (true) {
        const int a = tok_arc(p.sv_tok[ly.sv0 + i]);
        const int prev = p.sv_prev[ly.sv0 + i];
        if (a < 0) break;
        if (cnt >= ly.pathcap || prev < 0) {
            set_status(st, WFST_ECAPACITY);
            break;
        }
        const bool eps = p.g.arc_src[a] < 0;
        int fr = -1;
        if (!eps && j == 0) {
            set_status(st, WFST_ECAPACITY);
            break;
        }
        if (!eps) {
            fr = p.kept[ly.kept0 + j - 1];
            j--;
        }
        cnt++;
        p.path_arc[end - cnt] = a;
        p.path_frame[end - cnt] = fr;
        i = prev;
    }
    st.path_len = cnt;
}

// Lattice-beam pruning, one block per utterance, token sets from last to
// first.  e(j, s) is the extra cost of the best completion from node (j, s):
// at the last set e = fl(tot(s) - B); an arc from (j, s) with prefix cost p
// into (j', d) has ex = fl(fl(p - c_j'(d)) + e(j', d)), and e(j, s) is the
// minimum ex over its recorded out-arcs.  Epsilon arcs inside a set are
// iterated to their fixed point (the epsilon graph is acyclic).
__global__ __launch_bounds__(1024) void lattice_backward_kernel(Params p)
{
    __shared__ int sh_changed;
    __shared__ long long sh_cnt;
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    if (st.status != 0) return;
    const UttLayout &ly = p.lay[u];
    const int Tp = st.Tp;
    const float lb = p.lattice_beam;
    const float B = st.final_cost;
    const bool use_final = p.g.final_w != nullptr && st.reached_final;
    uint32_t *e = p.e_key + ly.sv0;
    const int64_t *so = p.sv_off + ly.fo0;
    const int64_t ntok = so[Tp + 1];
    const uint32_t kinf = okey(__int_as_float(0x7F800000));
    for (int64_t i = threadIdx.x; i < ntok; i += blockDim.x) e[i] = kinf;
    // Records were appended token set by token set, so the records of set j
    // are those whose source survivor lies in S_j: locate each set's range by
    // binary search on the source index.
    const int64_t ne = st.le_cnt, nx = st.lx_cnt;
    for (int j = threadIdx.x; j <= Tp + 1; j += blockDim.x) {
        const int64_t lo_sv = so[j];
        int64_t a = 0, b = ne;
        while (a < b) {
            int64_t mid = (a + b) >> 1;
            if (p.lat_e[ly.le0 + mid].x < lo_sv) a = mid + 1;
            else b = mid;
        }
        p.le_off[ly.fo0 + j] = a;
        a = 0;
        b = nx;
        while (a < b) {
            int64_t mid = (a + b) >> 1;
            if (p.lat_x[ly.lx0 + mid].x < lo_sv) a = mid + 1;
            else b = mid;
        }
        p.lx_off[ly.fo0 + j] = a;
    }
    __syncthreads();
    {
        const int64_t a = p.sv_off[ly.fo0 + Tp], b = p.sv_off[ly.fo0 + Tp + 1];
        for (int64_t i = a + threadIdx.x; i < b; i += blockDim.x) {
            int s = p.sv_state[ly.sv0 + i];
            float c = tok_cost(p.sv_tok[ly.sv0 + i]);
            float tot = c + (use_final ? p.g.final_w[s] : 0.0f);
            e[i] = okey(tot - B);
        }
    }
    __syncthreads();
    for (int j = Tp; j >= 0; j--) {
        if (threadIdx.x == 0) sh_cnt = 0;
        __syncthreads();
        long long kept = 0;
        if (j < Tp) {
            const int64_t r0 = p.le_off[ly.fo0 + j], r1 = p.le_off[ly.fo0 + j + 1];
            for (int64_t r = r0 + threadIdx.x; r < r1; r += blockDim.x) {
                int4 x = p.lat_e[ly.le0 + r];
                float cd = tok_cost(p.sv_tok[ly.sv0 + x.y]);
                float ed = okey_val(ld_relaxed(e + x.y));
                float d1 = __int_as_float(x.w) - cd;
                float ex = d1 + ed;
                p.ex_e[ly.le0 + r] = ex;
                atomicMin(e + x.x, okey(ex));
                kept += ex <= lb;
            }
        }
        __syncthreads();
        const int64_t q0 = p.lx_off[ly.fo0 + j], q1 = p.lx_off[ly.fo0 + j + 1];
        if (q1 > q0) {
            while (true) {
                if (threadIdx.x == 0) sh_changed = 0;
                __syncthreads();
                int changed = 0;
                for (int64_t r = q0 + threadIdx.x; r < q1; r += blockDim.x) {
                    int4 x = p.lat_x[ly.lx0 + r];
                    float cd = tok_cost(p.sv_tok[ly.sv0 + x.y]);
                    float ed = okey_val(ld_relaxed(e + x.y));
                    float d1 = __int_as_float(x.w) - cd;
                    float ex = d1 + ed;
                    p.ex_x[ly.lx0 + r] = ex;
                    uint32_t kx = okey(ex);
                    if (kx < ld_relaxed(e + x.x)) {
                        atomicMin(e + x.x, kx);
                        changed = 1;
                    }
                }
                if (changed) sh_changed = 1;
                __threadfence_block();
                __syncthreads();
                const int again = sh_changed;
                __syncthreads();
                if (!again) break;
            }
            for (int64_t r = q0 + threadIdx.x; r < q1; r += blockDim.x) kept += p.ex_x[ly.lx0 + r] <= lb;
        }
        kept = wave_sum_ll(kept);
        if (lane_id() == 0 && kept) atomicAdd(reinterpret_cast<unsigned long long *>(&sh_cnt), static_cast<unsigned long long>(kept));
        __syncthreads();
        if (threadIdx.x == 0) p.lo_off[ly.fo0 + j] = sh_cnt;
        __syncthreads();
    }
    // exclusive prefix over token sets -> output offsets
    if (threadIdx.x == 0) {
        int64_t run = 0;
        for (int j = 0; j <= Tp; j++) {
            int64_t c = p.lo_off[ly.fo0 + j];
            p.lo_off[ly.fo0 + j] = run;
            run += c;
        }
        p.lo_off[ly.fo0 + Tp + 1] = run;
        st.lat_kept = run;
    }
}

__device__ __forceinline__ void cas16(int4 *v, int i, int j)
{
    int4 a = v[i], b = v[j];
    if (b.y < a.y) {
        v[i] = b;
        v[j] = a;
    }
}

// Ascending sort of n records by arc id (unique within a token set): the
// bitonic network in its "flip" form, where every comparator puts the
// smaller key first, so positions >= n act as +inf and are never touched.
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

constexpr int kSortLds = 2048;

// One block per (token set j, utterance): gather the kept arcs of set j,
// sort them by arc and write {frame, arc, cost, extra}.
__global__ __launch_bounds__(256) void lattice_emit_kernel(Params p)
{
    __shared__ int4 buf[kSortLds];
    __shared__ int sh_n;
    const int u = blockIdx.y;
    const int j = blockIdx.x;
    UttState &st = p.st[u];
    if (st.status != 0 || j > st.Tp) return;
    const UttLayout &ly = p.lay[u];
    const float lb = p.lattice_beam;
    const int64_t o0 = p.lo_off[ly.fo0 + j];
    const int n = static_cast<int>(p.lo_off[ly.fo0 + j + 1] - o0);
    if (n == 0) return;
    int4 *out = p.lat_out + ly.lo0 + o0;
    const bool in_lds = n <= kSortLds;
    int4 *v = in_lds ? buf : out;
    if (threadIdx.x == 0) sh_n = 0;
    __syncthreads();
    for (int part = 0; part < 2; part++) {
        int64_t r0, r1;
        const int4 *rec;
        const float *ex;
        int64_t base;
        if (part == 0) {
            if (j == st.Tp) continue;
            r0 = p.le_off[ly.fo0 + j];
            r1 = p.le_off[ly.fo0 + j + 1];
            rec = p.lat_e;
            ex = p.ex_e;
            base = ly.le0;
        } else {
            r0 = p.lx_off[ly.fo0 + j];
            r1 = p.lx_off[ly.fo0 + j + 1];
            rec = p.lat_x;
            ex = p.ex_x;
            base = ly.lx0;
        }
        for (int64_t r = r0 + threadIdx.x; r < r1; r += blockDim.x) {
            float x = ex[base + r];
            if (x <= lb) {
                int slot = atomicAdd(&sh_n, 1);
                int4 q = rec[base + r];
                if (slot < n) v[slot] = make_int4(j, q.z, q.w, __float_as_int(x));
            }
        }
    }
    __syncthreads();
    sort_records(v, n);
    if (in_lds)
        for (int i = threadIdx.x; i < n; i += blockDim.x) out[i] = buf[i];
}

}  // namespace

hipError_t launch_final(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(final_kernel, dim3(p.U), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_backtrace(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(backtrace_kernel, dim3((p.U + 63) / 64), dim3(64), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_lattice_backward(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(lattice_backward_kernel, dim3(p.U), dim3(1024), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_lattice_emit(const Params &p, int max_frames, hipStream_t s)
{
    hipLaunchKernelGGL(lattice_emit_kernel, dim3(max_frames + 1, p.U), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace wfd
