// attn_fwd_bf16.hip -- bf16 instantiations of the single-pass attention
// forward (Eq. 3); the kernel is in attn_fwd_kernel.h.
#include "attn_fwd_kernel.h"

namespace sdattn {

hipError_t launch_attn_fwd_tiled_bf16(const AttnArgs& a) {
    using Seq = std::make_integer_sequence<int, 32>;   // D = 8, 16, ..., 256
    return dispatch_d<kBF16>(a, Seq{});
}

}  // namespace sdattn
