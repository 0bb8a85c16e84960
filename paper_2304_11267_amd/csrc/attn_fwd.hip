// attn_fwd.hip -- entry points of the single-pass attention forward (Eq. 3)
// and its fp16 instantiations; the kernel is in attn_fwd_kernel.h.
#include "attn_fwd_kernel.h"

namespace sdattn {

long long attn_fwd_grid(int B, int H, int Lq) {
    // the largest grid any geometry launches (32-row blocks bound it)
    return (long long)B * H * ((Lq + 31) / 32);
}

hipError_t launch_attn_fwd(const AttnArgs& a) {
    if (attn_fwd_short_supported(a.D, a.Lk)) return launch_attn_fwd_short(a);
    if (a.D < 32) return launch_attn_fwd_generic(a);
    if (a.dtype != kF16) return launch_attn_fwd_tiled_bf16(a);
    using Seq = std::make_integer_sequence<int, 32>;   // D = 8, 16, ..., 256
    return dispatch_d<kF16>(a, Seq{});
}

}  // namespace sdattn
