// attn_fwd_short.hip -- attention forward (Eq. 3) for short key sequences
// (Lk <= 128), the cross-attention over SD's 77-token text context.
//
// With at most two 64-key tiles, every key and value of a (batch, head) fits
// in LDS at once, so the kernel reads them a single time, computes the exact
// row maximum over all keys (no running maximum, no rescale of O) and then
// p and P V -- Eq. 4's reduction and the element-wise step in one pass over
// registers.  The work is bound by streaming Q in and O out of HBM; all loads
// are issued up front and awaited once.
//
// Operand layouts are those of the long-sequence kernel: S^T = K Q^T and
// O^T = V^T P^T on 32x32x16 MFMAs with one query per lane, V^T produced by
// ds_read_b64_tr_b16 from row-major V, and the row sum taken from a row of
// ones at d = D when D is not a multiple of 32.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kBQ = kWaves * 32;
constexpr int kKB = 64;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

template <int D, int NKT>
struct ShortGeom {
    static constexpr int DK = (D + 15) / 16;
    static constexpr int DN = (D + 31) / 32;
    static constexpr bool kOnes = (D % 32) != 0;
    static constexpr int kRows = NKT * kKB;                   // key rows held in LDS
    static constexpr int kBlockBytes = kRows * D * 2;         // K, V or the constant block
    static constexpr int kChunks = kBlockBytes / 1024;        // 1 KiB wave copies per block
    static constexpr int kLdsBytes = kBlockBytes * (kOnes ? 3 : 2);
};

__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    const int per = nblk / 8, rem = nblk % 8;
    const int xcd = bid % 8, slot = bid / 8;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

__device__ __forceinline__ u32x2 lds_read_tr(const char* p) {
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
    return __builtin_bit_cast(u32x2, v);
}

template <int ET, int D, int NKT>
__global__ __launch_bounds__(kThreads) void attn_fwd_short_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    uint16_t* __restrict__ O, float* __restrict__ LS, int Lq, int Lk, float scale_abs, float c,
    int neg, int nqb) {
    using G = ShortGeom<D, NKT>;
    constexpr int DK = G::DK;
    constexpr int DN = G::DN;
    constexpr int BB = G::kBlockBytes;

    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int bh = tile / nqb;
    const int qb = tile - bh * nqb;
    const int q0 = qb * kBQ + wave * 32;

    const char* Kh = (const char*)(K + (size_t)bh * Lk * D);
    const char* Vh = (const char*)(V + (size_t)bh * Lk * D);

    // All key rows of K and V (rows past Lk repeat row Lk - 1), 1 KiB per wave copy.
#pragma unroll
    for (int i = 0; i < (2 * G::kChunks + kWaves - 1) / kWaves; ++i) {
        const int cidx = wave + kWaves * i;
        if (cidx < 2 * G::kChunks) {
            const bool isv = cidx >= G::kChunks;
            const int cc = isv ? cidx - G::kChunks : cidx;
            const int byte = cc * 1024 + lane * 16;
            const int row = byte / (2 * D);
            const int col = byte - row * (2 * D);
            const size_t goff = (size_t)min(row, Lk - 1) * (2 * D) + col;
            __builtin_amdgcn_global_load_lds((isv ? Vh : Kh) + goff,
                                             (lds_void_t*)(smem + (isv ? BB : 0) + cc * 1024), 16, 0, 0);
        }
    }

    // Q^T operand: lane holds query q0 + l32, d = 16s + 8*half .. +7.
    const int qrow = q0 + l32;
    u32x4 qreg[DK];
#pragma unroll
    for (int s = 0; s < DK; ++s) {
        const int d0 = 16 * s + 8 * half;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (qrow < Lq && d0 < D) v = *(const u32x4*)(Q + ((size_t)bh * Lq + qrow) * D + d0);
        if (neg) v ^= 0x80008000u;
        qreg[s] = v;
    }

    // Constant block: a one in column 0 of every row (the row-sum column).
    if constexpr (G::kOnes) {
        const uint32_t one = from_float<ET>(1.0f);
        for (int i = tid; i < BB / 16; i += kThreads) {
            const int e0 = i * 8;   // first element of this 16-byte chunk
            u32x4 w = {0u, 0u, 0u, 0u};
            if (e0 % D == 0) w[0] = one;
            *(u32x4*)(smem + 2 * BB + i * 16) = w;
        }
    }

    const int k_off = (l32 * D + 8 * half) * 2;
    int v_off[DN];
    {
        const int g = lane >> 4, i = lane & 15;
        const int krow = 4 * (g >> 1) + (i >> 2);
#pragma unroll
        for (int n = 0; n < DN; ++n) {
            const int ds = 32 * n + 16 * (g & 1) + 4 * (i & 3);
            v_off[n] = ds < D ? BB + (krow * D + ds) * 2 : 2 * BB + (krow * D + ds - D) * 2;
        }
    }

    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // S^T for every key tile
    f32x16 st[NKT][2];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) st[kt][t][r] = 0.0f;
#pragma unroll
            for (int s = 0; s < DK; ++s) {
                const u32x4 a = *(const u32x4*)(smem + k_off + ((64 * kt + 32 * t) * D + 16 * s) * 2);
                st[kt][t] = mfma32x32x16<ET>(a, qreg[s], st[kt][t]);
            }
        }

    // exact row maximum over the keys < Lk
    float mloc = -__builtin_inff();
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = 64 * kt + 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                if (key < Lk) mloc = fmaxf(mloc, st[kt][t][r]);
            }
    const float s_max = half_max(mloc);
    const float negm = -(s_max * c);

    f32x16 acc[DN];
#pragma unroll
    for (int n = 0; n < DN; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[n][r] = 0.0f;
    float l_part = 0.0f;

#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
        u32x4 pk[2][2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            float p[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key = 64 * kt + 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                p[r] = key < Lk ? fast_exp2(fmaf(st[kt][t][r], c, negm)) : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w) pk[t][u][w] = pack2<ET>(p[8 * u + 2 * w], p[8 * u + 2 * w + 1]);
            if constexpr (!G::kOnes) {
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int w = 0; w < 4; ++w) l_part = add_pair<ET>(pk[t][u][w], l_part);
            }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int n = 0; n < DN; ++n) {
                    const char* vb = smem + v_off[n] + (64 * kt + 32 * t + 16 * u) * D * 2;
                    const u32x2 lo = lds_read_tr(vb);
                    const u32x2 hi = lds_read_tr(vb + 8 * D * 2);
                    const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                    acc[n] = mfma32x32x16<ET>(a, pk[t][u], acc[n]);
                }
    }

    float l;
    if constexpr (G::kOnes) {
        constexpr int dd = D % 32;
        constexpr int hsel = (dd >> 2) & 1, rsel = 4 * (dd >> 3) + (dd & 3);
        const float own = acc[D / 32][rsel];
        const float other = half_partner(own, half);
        l = (half == hsel) ? own : other;
    } else {
        l = half_sum(l_part);
    }
    const float inv = 1.0f / l;
    if (qrow < Lq) {
        uint16_t* orow = O + ((size_t)bh * Lq + qrow) * D;
#pragma unroll
        for (int n = 0; n < DN; ++n)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int d0 = 32 * n + 8 * g + 4 * half;
                if (d0 < D) {
                    u32x2 w;
                    w[0] = pack2<ET>(acc[n][4 * g + 0] * inv, acc[n][4 * g + 1] * inv);
                    w[1] = pack2<ET>(acc[n][4 * g + 2] * inv, acc[n][4 * g + 3] * inv);
                    *(u32x2*)(orow + d0) = w;
                }
            }
        if (LS && half == 0) {
            float* o2 = LS + ((size_t)bh * Lq + qrow) * 2;
            o2[0] = s_max * scale_abs;
            o2[1] = l;
        }
    }
}

template <int ET, int D, int NKT>
hipError_t launch_short_dn(const AttnArgs& a) {
    using G = ShortGeom<D, NKT>;
    const int nqb = (a.Lq + kBQ - 1) / kBQ;
    const long long nblk = (long long)a.B * a.H * nqb;
    const float scale_abs = a.scale < 0 ? -a.scale : a.scale;
    const float c = scale_abs * kLog2e;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&attn_fwd_short_kernel<ET, D, NKT>),
        hipFuncAttributeMaxDynamicSharedMemorySize, G::kLdsBytes);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL((attn_fwd_short_kernel<ET, D, NKT>), dim3((unsigned)nblk), dim3(kThreads),
                       G::kLdsBytes, (hipStream_t)a.stream, (const uint16_t*)a.q,
                       (const uint16_t*)a.k, (const uint16_t*)a.v, (uint16_t*)a.out, a.ls, a.Lq,
                       a.Lk, scale_abs, c, a.scale < 0 ? 1 : 0, nqb);
    return hipGetLastError();
}

template <int ET, int D>
hipError_t launch_short_d(const AttnArgs& a) {
    return a.Lk <= kKB ? launch_short_dn<ET, D, 1>(a) : launch_short_dn<ET, D, 2>(a);
}

template <int ET, int... Ds>
hipError_t dispatch_short(const AttnArgs& a, std::integer_sequence<int, Ds...>) {
    hipError_t r = hipErrorInvalidValue;
    bool hit = ((a.D == 32 + 8 * Ds ? (r = launch_short_d<ET, 32 + 8 * Ds>(a), true) : false) || ...);
    return hit ? r : hipErrorInvalidValue;
}

}  // namespace

bool attn_fwd_short_supported(int D, int Lk) {
    // D from 32 to 160 in steps of 8; LDS = 3 blocks of 128 key rows at most
    return Lk <= 2 * kKB && D >= 32 && D <= 160 && D % 8 == 0;
}

hipError_t launch_attn_fwd_short(const AttnArgs& a) {
    using Seq = std::make_integer_sequence<int, 17>;   // D = 32, 40, ..., 160
    return a.dtype == kF16 ? dispatch_short<kF16>(a, Seq{}) : dispatch_short<kBF16>(a, Seq{});
}

}  // namespace sdattn
