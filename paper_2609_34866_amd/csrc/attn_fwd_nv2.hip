// attn_fwd_nv2.hip -- the attention kernel with two value tensors per pass (the sweep's
// bit-width triples that share b_Q and b_K: one S^T and softmax, two outputs), in a
// translation unit of its own so the two halves of the attention build in parallel.
#include "attn_fwd_impl.h"

namespace jab {

template <int DT, int DH>
hipError_t run_attn_nv2(const AttnArgs &a, hipStream_t st) {
    return run_attn_cfg<DT, DH, 2, 1, 4>(a, st);
}

template hipError_t run_attn_nv2<F16, 16>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_nv2<F16, 64>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_nv2<F16, 128>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_nv2<BF16, 16>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_nv2<BF16, 64>(const AttnArgs &, hipStream_t);
template hipError_t run_attn_nv2<BF16, 128>(const AttnArgs &, hipStream_t);

}  // namespace jab
