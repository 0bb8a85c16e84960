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
// One launch may carry up to three independent products (the block's Q, K
// and V projections, whose inputs differ for cross-attention), each possibly
// a batch of equal-sized products at fixed strides (the 36 products of a
// Winograd convolution); each workgroup finds its product and batch item
// from its tile index, so the small context projections run beside the
// large latent one instead of after it.
//
// Workgroup tile: 128 token rows x 64 output channels, four waves of 32 rows.
// Each 64-channel slice of the x and w tiles is copied global -> LDS with
// global_load_lds (16 bytes per lane, whole 128-byte rows per instruction,
// no registers), into a ring of kStages slices so that kStages - 1 copies are
// in flight while one slice is multiplied.  Inside a slice, row r's 16-byte
// chunk c sits at chunk position c ^ swz(r), which keeps the MFMA operand
// reads (ds_read_b128, one row per lane) free of bank conflicts.  The product
// runs as y^T = w x^T on 32x32x16 MFMAs: A = 32 weight rows x 16 channels,
// B = 16 channels x 32 token rows, one token row per lane; each lane ends with
// 4 consecutive output channels per register group; the tile goes out through
// LDS so that each lane stores 16 contiguous bytes.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {


constexpr int kBM = 128;                          // token rows per workgroup
constexpr int kBN = 64;                           // output channels per workgroup
constexpr int kBK = 64;                           // input channels per slice
constexpr int kUnits = (kBM + kBN) * kBK / 8;     // 16-byte chunks per slice (1536)
constexpr int kSliceBytes = kUnits * 16;          // 24 KiB
constexpr int kCopies = kUnits / 64 / 4;          // copy instructions per wave per slice (6)
constexpr int kStages = 3;
constexpr int kLdsBytes = kStages * kSliceBytes;  // 72 KiB: two workgroups per CU

struct LinProblem {
    const uint16_t* x;
    const uint16_t* w;
    const uint16_t* bias;   // null: no bias
    uint16_t* y;
    int M, K, N, L;         // M = B*L token rows
    int xhw, yhw;           // head widths of the heads layouts (1 for rows layout)
    int nnt, tile0;         // channel tiles; first tile index of this product
    int per_batch;          // tiles of one batch item
    long long sx, sw, sy;   // element strides between batch items
};
struct LinGroup {
    LinProblem p[kMaxLinearProblems];
    int n;
};

// chunk-position swizzle of row r: distinct for any 8 consecutive rows, and
// (r & 1, swz) distinct for any 16 consecutive rows
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// c / hw for 0 <= c < 2^16 and 8 <= hw: the fp32 quotient is within one of
// the true one, and one correction step makes it exact.
__device__ __forceinline__ int div_small(int c, int hw, float inv_hw) {
    int h = (int)((float)c * inv_hw);
    h -= (h * hw > c) ? 1 : 0;
    h += ((h + 1) * hw <= c) ? 1 : 0;
    return h;
}

// Element offset of token row m = b*L + l (channel 0, head 0) in a tensor of
// C channels, and of channel c relative to it.
template <bool HEADS>
__device__ __forceinline__ size_t row_base(int m, int L, int C, int hw) {
    if constexpr (HEADS) {
        const int b = m / L, l = m - b * L;
        return ((size_t)b * (C / hw) * L + l) * hw;
    } else {
        return (size_t)m * C;
    }
}
template <bool HEADS>
__device__ __forceinline__ size_t chan_offset(int c, int L, int hw, float inv_hw) {
    if constexpr (HEADS) {
        const int h = div_small(c, hw, inv_hw);
        return (size_t)h * L * hw + (c - h * hw);
    } else {
        return (size_t)c;
    }
}

// Wait until at most `ahead` slices of this wave's copies are still in flight.
__device__ __forceinline__ void wait_slices(int ahead) {
    static_assert(kStages == 3, "wait_slices covers ahead = 0 and 1");
    if (ahead >= 1) __builtin_amdgcn_s_waitcnt(vm_wait(kCopies));
    else __builtin_amdgcn_s_waitcnt(vm_wait(0));
}

// Workgroup barrier after this wave's LDS reads have returned.  The slice
// copies are waited for explicitly (wait_slices); a fence here would drain
// every copy still in flight, since they count as LDS writes.  The memory
// clobber keeps the compiler from moving LDS reads across the barrier.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int ET, bool XH, bool YH>
__global__ __launch_bounds__(256) void linear_kernel(const LinGroup grp) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int pi = (grp.n > 2 && tile >= grp.p[2].tile0) ? 2 : (grp.n > 1 && tile >= grp.p[1].tile0) ? 1 : 0;
    const LinProblem& P = grp.p[pi];
    const int bi = (tile - P.tile0) / P.per_batch;     // batch item
    const int local = tile - P.tile0 - bi * P.per_batch;
    const uint16_t* __restrict__ X = P.x + bi * P.sx;
    const uint16_t* __restrict__ W = P.w + bi * P.sw;
    const int M = P.M, K = P.K, N = P.N, L = P.L, xhw = P.xhw;
    const int nt = local % P.nnt;        // consecutive workgroups share the token rows
    const int m0 = (local / P.nnt) * kBM;
    const int n0 = nt * kBN;
    const int nk = (K + kBK - 1) / kBK;

    // Copy j of this wave moves 16-byte chunk c of tile row r (x rows first,
    // then w rows); rows past M or N repeat the last row (their outputs are
    // never stored), channels past K repeat the last chunk (their operands are
    // zeroed before use).  Row bases are fixed across slices.
    size_t cbase[kCopies];
    int cch[kCopies];
#pragma unroll
    for (int j = 0; j < kCopies; ++j) {
        const int u0 = (wave * kCopies + j) * 64;
        const int u = u0 + lane;
        if (u0 < kBM * 8) {
            const int r = u >> 3;
            cch[j] = 8 * ((u & 7) ^ swz(r));
            cbase[j] = row_base<XH>(min(m0 + r, M - 1), L, K, xhw);
        } else {
            const int r = (u >> 3) - kBM;
            cch[j] = 8 * ((u & 7) ^ swz(r));
            cbase[j] = (size_t)min(n0 + r, N - 1) * K;
        }
    }
    const float inv_xhw = 1.0f / (float)xhw;

    // slice i (channels 64i .. 64i + 63) into ring slot i % kStages
    auto issue = [&](int i) __attribute__((always_inline)) {
        const int k0 = i * kBK;
        char* st = smem + (i % kStages) * kSliceBytes;
#pragma unroll
        for (int j = 0; j < kCopies; ++j) {
            const int u0 = (wave * kCopies + j) * 64;
            const int ch = min(k0 + cch[j], K - 8);
            const char* src = u0 < kBM * 8
                                  ? (const char*)(X + cbase[j] + chan_offset<XH>(ch, L, xhw, inv_xhw))
                                  : (const char*)(W + cbase[j] + ch);
            __builtin_amdgcn_global_load_lds(src, (lds_void_t*)(st + u0 * 16), 16, 0, 0);
        }
    };

    // operand offsets inside a slice: B = x row 32*wave + l32, A_t = w row
    // 32t + l32, chunk 2s + half for k-step s (rows 32t + l32 share swz(l32))
    const int hx = swz(l32);
    int offx[4], offw[2][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int cpos = (2 * s + half) ^ hx;
        offx[s] = ((32 * wave + l32) * 8 + cpos) * 16;
#pragma unroll
        for (int t = 0; t < 2; ++t) offw[t][s] = ((kBM + 32 * t + l32) * 8 + cpos) * 16;
    }

    // bias of this lane's output channels (8-byte aligned groups of 4),
    // fetched before the product
    const uint16_t* __restrict__ Bias = P.bias;
    u32x2 bias[2][4];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) bias[t][g] = u32x2{0u, 0u};
    if (Bias) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = min(n0 + 32 * t + 8 * g + 4 * half, N - 4);
                bias[t][g] = *(const u32x2*)(Bias + n);
            }
    }

    f32x16 acc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.0f;

#pragma unroll
    for (int i = 0; i < kStages - 1; ++i)
        if (i < nk) issue(i);

    for (int i = 0; i < nk; ++i) {
        wait_slices(min(nk - 1 - i, kStages - 2));
        lds_barrier();   // slice i is in LDS for every wave; slot (i - 1) % kStages is free
        if (i + kStages - 1 < nk) issue(i + kStages - 1);
        const char* st = smem + (i % kStages) * kSliceBytes;
        const int kval = K - i * kBK;    // channels of this slice inside K (uniform)
        // all twelve operand reads first, so their latencies overlap
        u32x4 bf[4], af[2][4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            bf[s] = *(const u32x4*)(st + offx[s]);
            af[0][s] = *(const u32x4*)(st + offw[0][s]);
            af[1][s] = *(const u32x4*)(st + offw[1][s]);
        }
        if (kval < kBK) {
#pragma unroll
            for (int s = 0; s < 4; ++s)
                if (8 * (2 * s + half) >= kval) {
                    bf[s] = u32x4{0u, 0u, 0u, 0u};
                    af[0][s] = bf[s];
                    af[1][s] = bf[s];
                }
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            acc[0] = mfma32x32x16<ET>(af[0][s], bf[s], acc[0]);
            acc[1] = mfma32x32x16<ET>(af[1][s], bf[s], acc[1]);
        }
    }

    // Stage the 128 x 64 output tile (bias added, rounded) in LDS, rows of
    // kOutStride bytes: lane (l32, half) holds channels 32t + 8g + 4*half + (0..3)
    // of tile row 32*wave + l32.
    constexpr int kOutStride = kBN * 2 + 16;
    static_assert(kBM * kOutStride <= kLdsBytes, "output tile fits in the slice ring");
    lds_barrier();   // every wave is done with the slices
    {
        char* orow = smem + (32 * wave + l32) * kOutStride;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = acc[t][4 * g + e] +
                           to_float<ET>((uint16_t)(bias[t][g][e >> 1] >> (16 * (e & 1))));
                u32x2 w;
                w[0] = pack2<ET>(v[0], v[1]);
                w[1] = pack2<ET>(v[2], v[3]);
                *(u32x2*)(orow + (32 * t + 8 * g + 4 * half) * 2) = w;
            }
    }
    lds_barrier();
    // 16 bytes per lane: chunk q = tid + 256j is tile row q / 8 + 32j, channels
    // n = n0 + 8 (q % 8) .. + 7 (inside one head, as head widths are multiples
    // of 8).  The channel offset is the same for all j; the row's batch and
    // token advance by 32 tokens per j.
    const int c8 = threadIdx.x & 7;
    const int n = n0 + 8 * c8;
    const int r0 = threadIdx.x >> 3;
    if (n < N) {
        const int yhw = P.yhw;
        uint16_t* __restrict__ Yc = P.y + bi * P.sy + chan_offset<YH>(n, L, yhw, 1.0f / (float)yhw);
        int b = (m0 + r0) / L, l = (m0 + r0) - b * L;   // token row m = b*L + l
#pragma unroll
        for (int j = 0; j < kBM * kBN / 8 / 256; ++j) {
            const int r = r0 + 32 * j;
            if (m0 + r < M) {
                const u32x4 v = *(const u32x4*)(smem + r * kOutStride + c8 * 16);
                const size_t row = YH ? ((size_t)b * (N / yhw) * L + l) * yhw : (size_t)(m0 + r) * N;
                *(u32x4*)(Yc + row) = v;
            }
            l += 32;
            while (l >= L) {
                l -= L;
                ++b;
            }
        }
    }
}

long long tiles_of(const LinearArgs& a) {
    return ((long long)a.B * a.L + kBM - 1) / kBM * ((a.N + kBN - 1) / kBN);
}

template <int ET, bool XH, bool YH>
hipError_t launch_t(const LinGroup& g, long long nblk, void* stream) {
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&linear_kernel<ET, XH, YH>),
        hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL((linear_kernel<ET, XH, YH>), dim3((unsigned)nblk), dim3(256), kLdsBytes,
                       (hipStream_t)stream, g);
    return hipGetLastError();
}

}  // namespace

long long linear_grid(int B, int L, int N) {
    LinearArgs a{};
    a.B = B;
    a.L = L;
    a.N = N;
    return tiles_of(a);
}

hipError_t launch_linear_group(const LinearArgs* a, int n) {
    if (n < 1 || n > kMaxLinearProblems) return hipErrorInvalidValue;
    LinGroup g{};
    long long nblk = 0;
    for (int i = 0; i < n; ++i) {
        if (a[i].dtype != a[0].dtype || a[i].x_heads != a[0].x_heads ||
            a[i].y_heads != a[0].y_heads || a[i].stream != a[0].stream)
            return hipErrorInvalidValue;
        LinProblem& p = g.p[i];
        p.x = (const uint16_t*)a[i].x;
        p.w = (const uint16_t*)a[i].w;
        p.bias = (const uint16_t*)a[i].bias;
        p.y = (uint16_t*)a[i].y;
        p.M = a[i].B * a[i].L;
        p.K = a[i].K;
        p.N = a[i].N;
        p.L = a[i].L;
        p.xhw = a[i].x_heads ? a[i].K / a[i].H : 1;
        p.yhw = a[i].y_heads ? a[i].N / a[i].H : 1;
        p.nnt = (a[i].N + kBN - 1) / kBN;
        p.tile0 = (int)nblk;
        p.per_batch = (int)tiles_of(a[i]);
        p.sx = a[i].sx;
        p.sw = a[i].sw;
        p.sy = a[i].sy;
        if (a[i].batch < 1) return hipErrorInvalidValue;
        nblk += tiles_of(a[i]) * a[i].batch;
        if (nblk > 0x7fffffff) return hipErrorInvalidValue;
    }
    g.n = n;
    if (nblk > 0x7fffffff) return hipErrorInvalidValue;
    const bool xh = a[0].x_heads, yh = a[0].y_heads;
    void* s = a[0].stream;
    if (a[0].dtype == kF16) {
        if (xh) return yh ? launch_t<kF16, true, true>(g, nblk, s) : launch_t<kF16, true, false>(g, nblk, s);
        return yh ? launch_t<kF16, false, true>(g, nblk, s) : launch_t<kF16, false, false>(g, nblk, s);
    }
    if (xh) return yh ? launch_t<kBF16, true, true>(g, nblk, s) : launch_t<kBF16, true, false>(g, nblk, s);
    return yh ? launch_t<kBF16, false, true>(g, nblk, s) : launch_t<kBF16, false, false>(g, nblk, s);
}

hipError_t launch_linear(const LinearArgs& a) { return launch_linear_group(&a, 1); }

}  // namespace sdattn
