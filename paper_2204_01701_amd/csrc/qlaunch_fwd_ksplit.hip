// qlaunch_fwd_ksplit.hip -- launch of the small-output forward kernel
// (qconv_fwd_ksplit.h).  Its own translation unit: it is compiled with the
// MFMA accumulators in VGPRs (build.py), which keeps them in place across the
// K loop where the AGPR form shuffled them through copies at one workgroup
// per CU.
#include "qhost.h"
#include "qconv_fwd_ksplit.h"

namespace ql {
namespace host {

template <typename T>
ql_status launch_fwd_ksplit(const FwdPlan &p, const FwdArgs &a, bool ep, hipStream_t st) {
    const dim3 grid((unsigned)(p.row_tiles * p.col_tiles));
#define QL_FWD_KSPLIT(RB, CB, NS)                                                                                \
    do {                                                                                                         \
        if (ep)                                                                                                  \
            hipLaunchKernelGGL((qconv_fwd_ksplit_kernel<T, RB, CB, NS, true>), grid, dim3(kThreads), 0, st, a);  \
        else                                                                                                     \
            hipLaunchKernelGGL((qconv_fwd_ksplit_kernel<T, RB, CB, NS, false>), grid, dim3(kThreads), 0, st, a); \
    } while (0)
    // ring stages per wave: two (two workgroups per CU; measured as fast or
    // faster on the 4 x 4 and 2 x 2 VGG-16 layers), or four (one per CU)
    const bool two = env_override("QLAYER_FWD_KSPLIT_NS", 2) != 4;
    if (p.krb == 2 && p.kcb == 4) {
        if (two) QL_FWD_KSPLIT(2, 4, 2);
        else QL_FWD_KSPLIT(2, 4, 4);
    } else if (p.krb == 1 && p.kcb == 4) {
        if (two) QL_FWD_KSPLIT(1, 4, 2);
        else QL_FWD_KSPLIT(1, 4, 4);
    } else if (p.krb == 2 && p.kcb == 2) {
        if (two) QL_FWD_KSPLIT(2, 2, 2);
        else QL_FWD_KSPLIT(2, 2, 4);
    } else {
        return QL_EINVAL;  // (the planner takes no other tile)
    }
#undef QL_FWD_KSPLIT
    return hip_status();
}

template ql_status launch_fwd_ksplit<uint16_t>(const FwdPlan &, const FwdArgs &, bool, hipStream_t);
template ql_status launch_fwd_ksplit<float>(const FwdPlan &, const FwdArgs &, bool, hipStream_t);

}  // namespace host
}  // namespace ql
