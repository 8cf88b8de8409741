// The search kernel without record workgroups (search_body.h), the frame
// classification that precedes it, and their launches.  The search kernel
// with record workgroups is instantiated in search_record_kernel.hip: a
// translation unit holding both instantiations compiles each of them into
// slower code (its arc-record gathers wait on LDS results one chunk at a
// time), so each has a file of its own.
#include "search_body.h"

namespace wfd {

namespace {

// isBlankFrame (Sec. 2, Alg. 1): frame t is blank when its blank
// log-likelihood exceeds the threshold (log domain); with a set of
// blank-like units (HMM topologies, Sec. 2) when any of them does.  Only
// every frame_stride-th frame is a candidate (a lower frame rate).  The kept
// frames are compacted in order, one workgroup per utterance.
__global__ __launch_bounds__(256) void classify_kernel(Params p)
{
    __shared__ int sh_scan[17];
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    const UttLayout &ly = p.lay[u];
    const int T = st.T;
    int base = 0;
    for (int t0 = 0; t0 < T; t0 += blockDim.x) {
        const int t = t0 + threadIdx.x;
        int keep = 0;
        if (t < T && t % p.frame_stride == 0) {
            const float *row = st.ll + static_cast<int64_t>(t) * p.L;
            keep = 1;
            for (int i = 0; i < p.n_blank; i++)
                if (row[p.blank_ids[i]] > p.blank_thr) keep = 0;
        }
        int total;
        const int ex = block_excl_scan(keep, sh_scan, &total);
        if (keep) p.kept[ly.kept0 + base + ex] = t;
        base += total;
    }
    if (threadIdx.x == 0) st.Tp = base;
}

}  // namespace

hipError_t launch_classify(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(classify_kernel, dim3(p.U), dim3(256), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_search(const Params &p, hipStream_t s)
{
    if (p.rec_wg > 0) return launch_search_record(p, s);
    hipLaunchKernelGGL(search_kernel<false>, dim3(p.U), dim3(kT), 0, s, p);
    return hipGetLastError();
}

}  // namespace wfd

