// The bf16 d = 128 instances of the two BoB pass launchers (and so of their
// kernels), in a translation unit of their own so that the build can give it
// LLVM's iterative ILP machine scheduler (-amdgpu-sched-strategy=
// iterative-ilp).  Measured on gfx950 against the default scheduler, in
// interleaved runs on one device: Pass 1 3.7% and Pass 2 2.2% faster at
// d = 128, while the same scheduler made the forward 34% and the first
// backward 13% slower, and the d = 64 Pass 2 7-8% and the d = 256 passes far
// slower, so every other kernel stays in flashbob.hip with the default.
#include "fb_launch.h"

namespace fb {

template int32_t launch_pass1<bf16, 128>(const Problem&, const void*, const void*, const void*, const void*,
                                         const void*, const void*, const void*, const void*, const float*,
                                         const float*, const void*, void*, void*, float*, float*, hipStream_t);
template int32_t launch_pass2<bf16, 128>(const Problem&, const void*, const void*, const void*, const void*,
                                         const void*, const void*, const void*, const float*, const float*,
                                         const float*, const float*, void*, void*, hipStream_t, const ColumnPlan&,
                                         float*);

}  // namespace fb
