// norm_act.hip -- the specialised kernels of Sec. 3.1: group normalisation
// (Eq. 1) in one launch with no intermediate tensor, and GELU (Eq. 2) fused
// with the split and multiply of the transformer's gated feed-forward.
//
// Group normalisation.  Feature maps are channel-major, [B, C, HW], so group
// (b, g) -- channels g*C/G .. (g+1)*C/G - 1 of batch b -- is one contiguous
// run of n = (C/G)*HW values.  A workgroup of 512 threads reads a group's
// run once into registers, 16 bytes per lane (n <= 49152 values: every UNet
// level, 40960 at 64x64 with 320 channels), and keeps it: the mean, then the
// mean square deviation from it (the two passes of the definition, over
// registers), then y = x*a_c + b_c with a_c = gamma_c / sqrt(var + eps) and
// b_c = beta_c - mean*a_c (gamma, beta staged in LDS).  With fewer than 256
// groups, S = 2 or 4 workgroups share a group, all on one XCD: each computes
// the statistics from the whole run (the later reads hit that XCD's L2) and
// writes 1/S of the output, so the launch covers the chip.  Larger groups
// (or pixel counts that are not a multiple of 8) take the same three steps
// in one workgroup, reading the run from memory each time.
//
// GEGLU.  h [M, 2F] -> out[m, f] = h[m, f] * GELU(h[m, F + f]); 16 bytes of
// each half per lane, one 16-byte store.  erf comes from the rational
// approximation 7.1.26 of Abramowitz and Stegun's Handbook of Mathematical
// Functions (absolute error below 1.5e-7), one exponential and one reciprocal
// per value.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

constexpr int kGnThreads = 512;
constexpr int kGnChunks = 12;                                 // 16-byte chunks per thread
constexpr long long kGnResident = (long long)kGnThreads * kGnChunks * 8;   // values
constexpr int kGnMaxCpg = 1024;   // channels per group the resident kernel stages

template <int ET>
__device__ __forceinline__ void unpack8(u32x4 v, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = to_float<ET>((uint16_t)(v[i] & 0xffffu));
        f[2 * i + 1] = to_float<ET>((uint16_t)(v[i] >> 16));
    }
}

template <int ET>
__device__ __forceinline__ u32x4 pack8(const float* f) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack2<ET>(f[2 * i], f[2 * i + 1]);
    return v;
}

// Sum of v over the workgroup (every thread gets it); red holds one float per wave.
__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    const int wave = threadIdx.x >> 6;
    __syncthreads();   // red is free (an earlier sum may still be read)
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    float s = 0.0f;
#pragma unroll
    for (int w = 0; w < kGnThreads / 64; ++w) s += red[w];
    return s;
}

template <int ET, int S>
__global__ __launch_bounds__(kGnThreads) void gn_resident_kernel(
    const uint16_t* X, const uint16_t* __restrict__ Gamma,
    const uint16_t* __restrict__ Beta, uint16_t* Y, int C, int HW, int G, int n, float eps,
    int ngroups) {
    __shared__ float red[kGnThreads / 64];
    __shared__ float gsh[kGnMaxCpg], bsh[kGnMaxCpg];   // the group's gamma and beta
    // S workgroups per group, all on one XCD (dispatch is round-robin over the
    // eight XCDs): each reads the whole group (the other S - 1 reads hit that
    // XCD's L2) and writes the s-th part of the output
    const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int bg = (slot / S) * 8 + xcd;
    const int sp = slot % S;
    if (bg >= ngroups) return;
    const int g = bg % G;
    const int cpg = C / G;
    const size_t base = (size_t)bg * n;
    const int nch = n / 8;
    const int tid = threadIdx.x;
    const int lo = (int)((long long)nch * sp / S), hi = (int)((long long)nch * (sp + 1) / S);
    for (int i = tid; i < cpg; i += kGnThreads) {   // read beside x; used after the statistics
        gsh[i] = Gamma ? to_float<ET>(Gamma[g * cpg + i]) : 1.0f;
        bsh[i] = Beta ? to_float<ET>(Beta[g * cpg + i]) : 0.0f;
    }

    u32x4 xr[kGnChunks];
#pragma unroll
    for (int j = 0; j < kGnChunks; ++j) {
        const int q = tid + kGnThreads * j;
        xr[j] = q < nch ? *(const u32x4*)(X + base + 8 * (size_t)q) : u32x4{0u, 0u, 0u, 0u};
    }
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < kGnChunks; ++j) {
        float f[8];
        unpack8<ET>(xr[j], f);
#pragma unroll
        for (int e = 0; e < 8; ++e) s += f[e];   // chunks past the run hold zeros
    }
    const float mean = block_sum(s, red) / (float)n;
    float s2 = 0.0f;
#pragma unroll
    for (int j = 0; j < kGnChunks; ++j) {
        if (tid + kGnThreads * j < nch) {
            float f[8];
            unpack8<ET>(xr[j], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float d = f[e] - mean;
                s2 = fmaf(d, d, s2);
            }
        }
    }
    const float var = block_sum(s2, red) / (float)n;
    const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
    for (int j = 0; j < kGnChunks; ++j) {
        const int q = tid + kGnThreads * j;
        if (q >= lo && q < hi) {
            const int cl = (8 * q) / HW;   // the chunk's channel in the group (HW % 8 == 0)
            const float a = rstd * gsh[cl];
            const float b = fmaf(-mean, a, bsh[cl]);
            float f[8];
            unpack8<ET>(xr[j], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) f[e] = fmaf(f[e], a, b);
            *(u32x4*)(Y + base + 8 * (size_t)q) = pack8<ET>(f);
        }
    }
}

// Any group size: the three steps each read the run from memory.  (X and Y
// may be the same tensor in both kernels: a group is read completely before
// its first value is written, and no other workgroup touches it.)
template <int ET>
__global__ __launch_bounds__(kGnThreads) void gn_generic_kernel(
    const uint16_t* X, const uint16_t* __restrict__ Gamma,
    const uint16_t* __restrict__ Beta, uint16_t* Y, int C, long long HW, int G, long long n,
    float eps) {
    __shared__ float red[kGnThreads / 64];
    const int bg = blockIdx.x;
    const int g = bg % G;
    const int cpg = C / G;
    const uint16_t* xg = X + (size_t)bg * n;
    uint16_t* yg = Y + (size_t)bg * n;
    float s = 0.0f;
    for (long long i = threadIdx.x; i < n; i += kGnThreads) s += to_float<ET>(xg[i]);
    const float mean = block_sum(s, red) / (float)n;
    float s2 = 0.0f;
    for (long long i = threadIdx.x; i < n; i += kGnThreads) {
        const float d = to_float<ET>(xg[i]) - mean;
        s2 = fmaf(d, d, s2);
    }
    const float var = block_sum(s2, red) / (float)n;
    const float rstd = 1.0f / sqrtf(var + eps);
    // every read of this group is done before the first write (y may be x)
    __syncthreads();
    for (long long i = threadIdx.x; i < n; i += kGnThreads) {
        const int c = g * cpg + (int)(i / HW);
        const float ga = Gamma ? to_float<ET>(Gamma[c]) : 1.0f;
        const float be = Beta ? to_float<ET>(Beta[c]) : 0.0f;
        yg[i] = from_float<ET>((to_float<ET>(xg[i]) - mean) * rstd * ga + be);
    }
}

// erf(x) by Abramowitz and Stegun 7.1.26: for x >= 0,
// erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-x^2), t = 1 / (1 + p x);
// erf is odd.
__device__ __forceinline__ float erf_as(float x) {
    const float ax = fabsf(x);
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
    float poly = 1.061405429f;
    poly = fmaf(poly, t, -1.453152027f);
    poly = fmaf(poly, t, 1.421413741f);
    poly = fmaf(poly, t, -0.284496736f);
    poly = fmaf(poly, t, 0.254829592f);
    const float e = fast_exp2(-ax * ax * kLog2e);
    const float r = fmaf(-poly * t, e, 1.0f);
    return copysignf(r, x);
}

// GELU (Eq. 2): x/2 (1 + erf(x / sqrt 2))
__device__ __forceinline__ float gelu(float x) {
    return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f));
}

template <int ET>
__global__ __launch_bounds__(256) void geglu_kernel(const uint16_t* __restrict__ H,
                                                    uint16_t* __restrict__ Out, long long total,
                                                    int F) {
    const int f8 = F / 8;   // 16-byte chunks per output row
    for (long long q = (long long)blockIdx.x * 256 + threadIdx.x; q < total;
         q += (long long)gridDim.x * 256) {
        const long long m = q / f8;
        const int c = (int)(q - m * f8);
        const uint16_t* hr = H + (size_t)m * 2 * F + 8 * c;
        const u32x4 av = *(const u32x4*)hr;
        const u32x4 gv = *(const u32x4*)(hr + F);
        float a[8], gt[8];
        unpack8<ET>(av, a);
        unpack8<ET>(gv, gt);
#pragma unroll
        for (int e = 0; e < 8; ++e) a[e] *= gelu(gt[e]);
        *(u32x4*)(Out + (size_t)m * F + 8 * c) = pack8<ET>(a);
    }
}

template <int ET>
hipError_t launch_gn_e(const GroupNormArgs& a) {
    const long long n = (long long)(a.C / a.G) * a.HW;
    const unsigned grid = (unsigned)(a.B * a.G);
    if (a.HW % 8 == 0 && n <= kGnResident && a.C / a.G <= kGnMaxCpg) {
        // several workgroups per group when there are few groups, unless in place
        const int ng = a.B * a.G;
        const int S = (ng >= 256 || a.x == a.y) ? 1 : ng >= 128 ? 2 : 4;
        const unsigned grid8 = (unsigned)((ng + 7) / 8 * 8 * S);
        auto k = S == 1 ? gn_resident_kernel<ET, 1> : S == 2 ? gn_resident_kernel<ET, 2> : gn_resident_kernel<ET, 4>;
        hipLaunchKernelGGL(k, dim3(grid8), dim3(kGnThreads), 0, (hipStream_t)a.stream,
                           (const uint16_t*)a.x, (const uint16_t*)a.gamma, (const uint16_t*)a.beta,
                           (uint16_t*)a.y, a.C, (int)a.HW, a.G, (int)n, a.eps, ng);
    } else {
        hipLaunchKernelGGL(gn_generic_kernel<ET>, dim3(grid), dim3(kGnThreads), 0,
                           (hipStream_t)a.stream, (const uint16_t*)a.x, (const uint16_t*)a.gamma,
                           (const uint16_t*)a.beta, (uint16_t*)a.y, a.C, a.HW, a.G, n, a.eps);
    }
    return hipGetLastError();
}

template <int ET>
hipError_t launch_geglu_e(const GegluArgs& a) {
    const long long total = a.M * (a.F / 8);
    const long long want = (total + 255) / 256;
    const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(geglu_kernel<ET>, dim3(grid), dim3(256), 0, (hipStream_t)a.stream,
                       (const uint16_t*)a.h, (uint16_t*)a.out, total, a.F);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_group_norm(const GroupNormArgs& a) {
    return a.dtype == kF16 ? launch_gn_e<kF16>(a) : launch_gn_e<kBF16>(a);
}

hipError_t launch_geglu(const GegluArgs& a) {
    return a.dtype == kF16 ? launch_geglu_e<kF16>(a) : launch_geglu_e<kBF16>(a);
}

}  // namespace sdattn
