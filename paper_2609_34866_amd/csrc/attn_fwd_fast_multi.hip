// attn_fwd_fast_multi.hip -- the fast attention kernel with two or four value tensors per pass (the
// sweep's triples that share b_Q and b_K: one score matrix and softmax, several outputs).  A
// translation unit of its own, built with the accumulators in the accumulation registers (one wave
// per SIMD: the output accumulators of the value tensors take 128 registers, the rest go to the
// score, key and value fragments).  Head_dim 128 takes two value tensors per pass: four would need
// 256 accumulators besides the fragments.
#include "attn_fwd_impl.h"
#include "attn_fwd_fast.h"

namespace jab {

template <int DT, int DH, int NV>
hipError_t run_attn_fast_multi(const AttnArgs &a, hipStream_t st) {
    static_assert(NV == 2 || NV == 4, "value tensors per pass");
    return launch_attn_fast<DT, DH, NV>(a, st);
}

template hipError_t run_attn_fast_multi<F16, 64, 2>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<F16, 64, 4>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<F16, 128, 2>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<F16, 128, 4>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<BF16, 64, 2>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<BF16, 64, 4>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<BF16, 128, 2>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_fast_multi<BF16, 128, 4>(const AttnArgs &, hipStream_t);

}  // namespace jab
