// The search kernel with record workgroups appended to its launch
// (search_body.h), in a translation unit of its own (see search_kernel.hip).
#include "search_body.h"

namespace wfd {

hipError_t launch_search_record(const Params &p, hipStream_t s)
{
    // the record workgroups wait on the search's published counts
    if (p.rec_wg <= 0 || p.U > kRecMaxUtts || p.pub_k <= 0 || !p.prog || !p.rec_next) return hipErrorInvalidValue;
    hipLaunchKernelGGL(search_kernel<true>, dim3(p.U + p.rec_wg), dim3(kT), 0, s, p);
    return hipGetLastError();
}

}  // namespace wfd
