// linear.hip -- the projections around the attention in SD's transformer
// blocks: y = x w^T + bias with weights stored [out, in], and the head
// split / merge folded into the addressing of the rows.
//
// A token row m = b*L + l of x (or y) lives either in rows layout [B, L, C]
// or in heads layout [B, H, L, C/H] (channel c = h*(C/H) + d at
// ((b*H + h)*L + l)*(C/H) + d).  Writing Q, K and V in heads layout is the
// head split before Eq. 3; reading O in heads layout is the head merge before
// the output projection -- neither needs a transpose of its own.
//
// The product runs as y^T = w x^T on 32x32x16 MFMAs with one token row per
// lane (as S^T = K Q^T in the attention kernels): A = 32 weight rows x 16
// input channels, B = 16 input channels x 32 token rows, both loaded 16 bytes
// per lane straight from global memory, and each lane ends with 4 consecutive
// output channels per register group, stored 8 bytes at a time.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

constexpr int kLinM = 128;   // token rows per workgroup (4 waves x 32)
constexpr int kLinN = 64;    // output channels per workgroup (2 MFMA tiles)
constexpr int kLinK = 64;    // input channels per loop step (4 MFMA k-steps)

__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    const int per = nblk / 8, rem = nblk % 8;
    const int xcd = bid % 8, slot = bid / 8;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Element offset of channel c of token row m = b*L + l in a tensor of C channels.
template <bool HEADS>
__device__ __forceinline__ size_t row_offset(int m, int c, int L, int C, int hw) {
    if constexpr (HEADS) {
        const int b = m / L, l = m - b * L;
        const int h = c / hw, d = c - h * hw;
        return ((size_t)(b * (C / hw) + h) * L + l) * hw + d;
    } else {
        return (size_t)m * C + c;
    }
}

template <int ET, bool XH, bool YH, bool BIAS>
__global__ __launch_bounds__(256) void linear_kernel(const uint16_t* __restrict__ X,
                                                     const uint16_t* __restrict__ W,
                                                     const uint16_t* __restrict__ Bias,
                                                     uint16_t* __restrict__ Y, int M, int K, int N,
                                                     int L, int xhw, int yhw, int nmt, int nnt) {
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int nt = tile % nnt;          // consecutive workgroups share the token rows
    const int mt = tile / nnt;
    const int m = mt * kLinM + wave * 32 + l32;      // this lane's token row
    const int n0 = nt * kLinN;
    const bool mvalid = m < M;
    const int ms = mvalid ? m : 0;

    // operands of one 16-channel k-step at input channel k: x[m][k + 8*half ..]
    // and w[n0 + 32t + l32][k + 8*half ..]; zero past K, N or M
    auto load_x = [&](int k) __attribute__((always_inline)) -> u32x4 {
        const int c = k + 8 * half;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (c < K && mvalid) v = *(const u32x4*)(X + row_offset<XH>(ms, c, L, K, xhw));
        return v;
    };
    auto load_w = [&](int k, int t) __attribute__((always_inline)) -> u32x4 {
        const int c = k + 8 * half;
        const int n = n0 + 32 * t + l32;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (c < K && n < N) v = *(const u32x4*)(W + (size_t)n * K + c);
        return v;
    };

    f32x16 acc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;

    constexpr int S = kLinK / 16;
    u32x4 xa[S], wa[S][2];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        xa[s] = load_x(16 * s);
        wa[s][0] = load_w(16 * s, 0);
        wa[s][1] = load_w(16 * s, 1);
    }
    for (int k0 = 0; k0 < K; k0 += kLinK) {
        u32x4 xb[S], wb[S][2];
        const bool more = k0 + kLinK < K;
        if (more) {   // next step's operands while this step's MFMAs run
#pragma unroll
            for (int s = 0; s < S; ++s) {
                xb[s] = load_x(k0 + kLinK + 16 * s);
                wb[s][0] = load_w(k0 + kLinK + 16 * s, 0);
                wb[s][1] = load_w(k0 + kLinK + 16 * s, 1);
            }
        }
#pragma unroll
        for (int s = 0; s < S; ++s)
#pragma unroll
            for (int t = 0; t < 2; ++t) acc[t] = mfma32x32x16<ET>(wa[s][t], xa[s], acc[t]);
        if (more) {
#pragma unroll
            for (int s = 0; s < S; ++s) {
                xa[s] = xb[s];
                wa[s][0] = wb[s][0];
                wa[s][1] = wb[s][1];
            }
        }
    }

    // output channels n0 + 32t + 8g + 4*half + (0..3) of token row m
    if (!mvalid) return;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = n0 + 32 * t + 8 * g + 4 * half;
            if (n < N) {   // N % 8 == 0: the 4 channels are all inside N and inside one head
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    v[e] = acc[t][4 * g + e];
                    if constexpr (BIAS) v[e] += to_float<ET>(Bias[n + e]);
                }
                u32x2 w;
                w[0] = pack2<ET>(v[0], v[1]);
                w[1] = pack2<ET>(v[2], v[3]);
                *(u32x2*)(Y + row_offset<YH>(m, n, L, N, yhw)) = w;
            }
        }
}

template <int ET, bool XH, bool YH, bool BIAS>
hipError_t launch_linear_t(const LinearArgs& a) {
    const int M = a.B * a.L;
    const int nmt = (M + kLinM - 1) / kLinM;
    const int nnt = (a.N + kLinN - 1) / kLinN;
    const long long nblk = (long long)nmt * nnt;
    hipLaunchKernelGGL((linear_kernel<ET, XH, YH, BIAS>), dim3((unsigned)nblk), dim3(256), 0,
                       (hipStream_t)a.stream, (const uint16_t*)a.x, (const uint16_t*)a.w,
                       (const uint16_t*)a.bias, (uint16_t*)a.y, M, a.K, a.N, a.L,
                       a.x_heads ? a.K / a.H : 1, a.y_heads ? a.N / a.H : 1, nmt, nnt);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_linear_e(const LinearArgs& a) {
    const bool b = a.bias != nullptr;
    if (a.x_heads) {
        if (a.y_heads) return b ? launch_linear_t<ET, true, true, true>(a) : launch_linear_t<ET, true, true, false>(a);
        return b ? launch_linear_t<ET, true, false, true>(a) : launch_linear_t<ET, true, false, false>(a);
    }
    if (a.y_heads) return b ? launch_linear_t<ET, false, true, true>(a) : launch_linear_t<ET, false, true, false>(a);
    return b ? launch_linear_t<ET, false, false, true>(a) : launch_linear_t<ET, false, false, false>(a);
}

}  // namespace

long long linear_grid(int B, int L, int N) {
    return ((long long)B * L + kLinM - 1) / kLinM * ((N + kLinN - 1) / kLinN);
}

hipError_t launch_linear(const LinearArgs& a) {
    return a.dtype == kF16 ? launch_linear_e<kF16>(a) : launch_linear_e<kBF16>(a);
}

}  // namespace sdattn
