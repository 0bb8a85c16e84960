// launch.h -- host-side launchers of the sdattn kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>

namespace sdattn {

struct AttnArgs {
    const void* q;
    const void* k;
    const void* v;
    void* out;
    float* ls;      // optional [B,H,Lq,2] (L, S), may be null
    int B, H, Lq, Lk, D;
    float scale;
    int dtype;      // ElemType: kF16 or kBF16
    void* stream;
    int o_rows = 0; // nonzero: out is [B, Lq, H*D] (heads merged) instead of [B, H, Lq, D]
};

// Number of workgroups the attention kernels launch for these sizes.
long long attn_fwd_grid(int B, int H, int Lq);
// Picks the kernel for (D, Lk) and launches it.
hipError_t launch_attn_fwd(const AttnArgs& a);
// the bf16 instantiations of the tiled kernel (a translation unit of their own)
hipError_t launch_attn_fwd_tiled_bf16(const AttnArgs& a);
// The generic kernel (any D % 8 == 0 up to 256).
hipError_t launch_attn_fwd_generic(const AttnArgs& a);
// The short-sequence kernel (all keys resident in LDS): Lk <= 128, 32 <= D <= 160.
bool attn_fwd_short_supported(int D, int Lk);
hipError_t launch_attn_fwd_short(const AttnArgs& a);

struct SoftmaxArgs {
    const void* a;
    float* ls;      // [rows, 2]
    void* p;        // optional [rows, cols], may be null
    long long rows, cols;
    float scale;
    int dtype;      // ElemType: kF16, kBF16 or kF32
    void* stream;
};

hipError_t launch_softmax_rows(const SoftmaxArgs& a);

// The first and last steps of the partially fused softmax (twopass.hip).
struct LogitsArgs {
    const void* q;
    const void* k;
    void* a;        // [B,H,Lq,Lk] of a_dtype
    int B, H, Lq, Lk, D;
    float scale;
    int dtype;      // Q, K: kF16 or kBF16
    int a_dtype;    // kF16, kBF16 or kF32
    void* stream;
};
long long logits_grid(int B, int H, int Lq, int Lk);
hipError_t launch_logits(const LogitsArgs& a);

struct SoftmaxPvArgs {
    const void* a;  // [B,H,Lq,Lk] of a_dtype
    const float* ls;   // [B,H,Lq,2] (L, S) of A's rows
    const void* v;
    void* out;
    int B, H, Lq, Lk, D;
    int dtype;      // V, out: kF16 or kBF16
    int a_dtype;    // kF16, kBF16 or kF32
    void* stream;
};
hipError_t launch_softmax_pv(const SoftmaxPvArgs& a);

// The projections around the attention (linear.hip).
struct LinearArgs {
    const void* x;
    const void* w;      // [N, K]
    const void* bias;   // [N] or null
    void* y;
    int B, L, K, N, H;
    bool x_heads, y_heads;   // [B, H, L, C/H] instead of [B, L, C]
    int dtype;
    void* stream;
    int batch = 1;           // independent products with the same sizes,
    long long sx = 0, sw = 0, sy = 0;   // element strides between their x, w and y
};
long long linear_grid(int B, int L, int N);
hipError_t launch_linear(const LinearArgs& a);
// Up to kMaxLinearProblems products of one element type and one pair of
// layouts in a single launch (e.g. the Q, K and V projections).
constexpr int kMaxLinearProblems = 3;
hipError_t launch_linear_group(const LinearArgs* a, int n);

// Group normalisation and GEGLU (norm_act.hip).
struct GroupNormArgs {
    const void* x;        // [B, C, HW]
    const void* gamma;    // [C] or null
    const void* beta;     // [C] or null
    void* y;              // like x (may be x)
    int B, C;
    long long HW;
    int G;
    float eps;
    int dtype;
    void* stream;
};
hipError_t launch_group_norm(const GroupNormArgs& a);

struct GegluArgs {
    const void* h;        // [M, 2F]
    void* out;            // [M, F]
    long long M;
    int F;                // multiple of 8
    int dtype;
    void* stream;
};
hipError_t launch_geglu(const GegluArgs& a);

// Winograd F(4x4, 3x3) convolution (winograd.hip).
struct WinoFilterArgs {
    const void* w;        // [Co, Ci, 3, 3]
    void* u;              // [36, Co, Ci]
    int Co, Ci;
    int dtype;
    void* stream;
};
struct WinoConvArgs {
    const void* x;        // [B, Ci, H, W]
    const void* u;        // [36, Co, Ci]
    const void* bias;     // [Co] or null
    void* y;              // [B, Co, H, W]
    void* v;              // [36, T, Ci] workspace
    void* m;              // [36, T, Co] workspace
    int B, Ci, Co, H, W;
    int dtype;
    void* stream;
};
long long wino_tiles(int B, int H, int W);
hipError_t launch_wino_filter(const WinoFilterArgs& a);
hipError_t launch_wino_conv(const WinoConvArgs& a);

}  // namespace sdattn
