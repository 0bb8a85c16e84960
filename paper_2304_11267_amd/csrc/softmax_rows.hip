// softmax_rows.hip -- Eq. 4's reduction (L, S) over the rows of a matrix, and
// optionally the element-wise step p = exp(a - L) / S, in one launch.
//
// Sec. 3.2.1 observes that mapping A to the N x 2 pair (L, S) has little
// parallelism and splits each row's reduction into stages over blocks of
// elements.  Here the stages are:
//   1. each lane folds its 16-byte chunks of the row into a running pair
//      (m, s) -- one rescale per chunk, one exponential per element;
//   2. the 64 lanes of a wave merge their pairs with a butterfly;
//   3. for long rows, the 4 waves of the workgroup each own a quarter of the
//      row and merge their pairs through LDS.
// Two pairs merge as (m, s) + (m', s') = (M, s e^{m-M} + s' e^{m'-M}),
// M = max(m, m'), which is exact in real arithmetic and order-free.
// The optional second pass re-reads the row (now in L2) and writes p.
//
// Rows of at most 64 * 16 chunks whose p is wanted (and short rows) take a
// register-resident variant: a wave
// holds its whole row (R chunks per lane, all loads issued at once), takes
// the exact maximum (stage 1 in the lane, stage 2 across the wave), then the
// sum of the exponentials the same way, and writes p from the exponentials it
// already holds -- the row is read from memory once.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

constexpr int kThreads = 256;
constexpr long long kMaxGrid = 1 << 20;

template <int ET>
struct Elem;
template <>
struct Elem<kF16> { static constexpr int kPerChunk = 8; };
template <>
struct Elem<kBF16> { static constexpr int kPerChunk = 8; };
template <>
struct Elem<kF32> { static constexpr int kPerChunk = 4; };

template <int ET>
__device__ __forceinline__ void load_chunk(const void* base, long long idx, float* x) {
    const u32x4 w = *((const u32x4*)base + idx);
    if constexpr (ET == kF32) {
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(w[e]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[2 * e] = to_float<ET>((uint16_t)(w[e] & 0xffffu));
            x[2 * e + 1] = to_float<ET>((uint16_t)(w[e] >> 16));
        }
    }
}

template <int ET>
__device__ __forceinline__ void store_chunk(void* base, long long idx, const float* x) {
    u32x4 w;
    if constexpr (ET == kF32) {
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(x[e]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = pack2<ET>(x[2 * e], x[2 * e + 1]);
    }
    *((u32x4*)base + idx) = w;
}

template <int ET>
__device__ __forceinline__ float load_one(const void* base, long long idx) {
    if constexpr (ET == kF32) return ((const float*)base)[idx];
    else return to_float<ET>(((const uint16_t*)base)[idx]);
}

template <int ET>
__device__ __forceinline__ void store_one(void* base, long long idx, float x) {
    if constexpr (ET == kF32) ((float*)base)[idx] = x;
    else ((uint16_t*)base)[idx] = from_float<ET>(x);
}

// weight of a partial sum taken at maximum m when the merged maximum is M
__device__ __forceinline__ float rescale_weight(float m, float M) {
    return m == M ? 1.0f : fast_exp2((m - M) * kLog2e);
}

__device__ __forceinline__ void merge_pair(float& m, float& s, float m2, float s2) {
    const float M = fmaxf(m, m2);
    s = s * rescale_weight(m, M) + s2 * rescale_weight(m2, M);
    m = M;
}

// WPR = waves per row (1 or 4); VEC = rows are read in 16-byte chunks.
template <int ET, int WPR, bool VEC>
__global__ __launch_bounds__(kThreads) void softmax_rows_kernel(
    const void* __restrict__ A, float* __restrict__ LS, void* __restrict__ P, long long rows,
    long long cols, float scale, long long ngroups) {
    constexpr int RPW = 4 / WPR;                 // rows per workgroup
    constexpr int EPC = VEC ? Elem<ET>::kPerChunk : 1;
    __shared__ float red[4][2];

    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int part = wave % WPR;
    const long long nunits = cols / EPC;          // chunks (or elements) per row
    const long long stride = 64LL * WPR;

    for (long long g = blockIdx.x; g < ngroups; g += gridDim.x) {
        const long long row = g * RPW + wave / WPR;
        const bool live = row < rows;
        float m = -__builtin_inff(), s = 0.0f;
        if (live) {
            const long long base = row * nunits;
            for (long long u = part * 64 + lane; u < nunits; u += stride) {
                float x[EPC];
                if constexpr (VEC) load_chunk<ET>(A, base + u, x);
                else x[0] = load_one<ET>(A, base + u);
                float cm = x[0] * scale;
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    x[e] *= scale;
                    cm = fmaxf(cm, x[e]);
                }
                const float mn = fmaxf(m, cm);
                const float nb = -mn * kLog2e;
                float acc = s * rescale_weight(m, mn);
#pragma unroll
                for (int e = 0; e < EPC; ++e) acc += fast_exp2(fmaf(x[e], kLog2e, nb));
                s = acc;
                m = mn;
            }
        }
        // stage 2: merge across the wave
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const float m2 = __shfl_xor(m, off);
            const float s2 = __shfl_xor(s, off);
            merge_pair(m, s, m2, s2);
        }
        // stage 3: merge the waves that share a row
        if constexpr (WPR > 1) {
            if (lane == 0) {
                red[wave][0] = m;
                red[wave][1] = s;
            }
            __syncthreads();
            const int w0 = wave - part;
            m = red[w0][0];
            s = red[w0][1];
#pragma unroll
            for (int w = 1; w < WPR; ++w) merge_pair(m, s, red[w0 + w][0], red[w0 + w][1]);
            __syncthreads();
        }
        if (live) {
            if (part == 0 && lane == 0) {
                LS[2 * row] = m;
                LS[2 * row + 1] = s;
            }
            if (P) {
                const float nb = -m * kLog2e;
                const float inv = 1.0f / s;
                const long long base = row * nunits;
                for (long long u = part * 64 + lane; u < nunits; u += stride) {
                    float x[EPC];
                    if constexpr (VEC) load_chunk<ET>(A, base + u, x);
                    else x[0] = load_one<ET>(A, base + u);
#pragma unroll
                    for (int e = 0; e < EPC; ++e) x[e] = fast_exp2(fmaf(x[e] * scale, kLog2e, nb)) * inv;
                    if constexpr (VEC) store_chunk<ET>(P, base + u, x);
                    else store_one<ET>(P, base + u, x[0]);
                }
            }
        }
    }
}

// One row per wave, held in registers: R chunks per lane (64 * R >= chunks).
template <int ET, int R>
__global__ __launch_bounds__(kThreads) void softmax_rows_reg_kernel(
    const void* __restrict__ A, float* __restrict__ LS, void* __restrict__ P, long long rows,
    long long cols, float scale, long long ngroups) {
    constexpr int EPC = Elem<ET>::kPerChunk;
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    const int nunits = (int)(cols / EPC);

    for (long long g = blockIdx.x; g < ngroups; g += gridDim.x) {
        const long long row = g * 4 + wave;
        if (row >= rows) continue;   // no barriers below: waves are independent
        const long long base = row * nunits;
        float x[R][EPC];
#pragma unroll
        for (int i = 0; i < R; ++i) {
            if (lane + 64 * i < nunits) load_chunk<ET>(A, base + lane + 64 * i, x[i]);
        }
        // exact row maximum of scale * a
        float m = -__builtin_inff();
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (lane + 64 * i < nunits) {
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    x[i][e] *= scale;
                    m = fmaxf(m, x[i][e]);
                }
            }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
        // exponentials (kept for p) and their sum
        const float nb = -m * kLog2e;
        float s = 0.0f;
#pragma unroll
        for (int i = 0; i < R; ++i)
            if (lane + 64 * i < nunits) {
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    x[i][e] = fast_exp2(fmaf(x[i][e], kLog2e, nb));
                    s += x[i][e];
                }
            }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
        if (lane == 0) {
            LS[2 * row] = m;
            LS[2 * row + 1] = s;
        }
        if (P) {
            const float inv = 1.0f / s;
#pragma unroll
            for (int i = 0; i < R; ++i)
                if (lane + 64 * i < nunits) {
#pragma unroll
                    for (int e = 0; e < EPC; ++e) x[i][e] *= inv;
                    store_chunk<ET>(P, base + lane + 64 * i, x[i]);
                }
        }
    }
}

template <int ET, int R>
hipError_t launch_reg(const SoftmaxArgs& a) {
    const long long ngroups = (a.rows + 3) / 4;
    const long long grid = ngroups < kMaxGrid ? ngroups : kMaxGrid;
    hipLaunchKernelGGL((softmax_rows_reg_kernel<ET, R>), dim3((unsigned)grid), dim3(kThreads), 0,
                       (hipStream_t)a.stream, a.a, a.ls, a.p, a.rows, a.cols, a.scale, ngroups);
    return hipGetLastError();
}

template <int ET, int WPR, bool VEC>
hipError_t launch3(const SoftmaxArgs& a) {
    constexpr int RPW = 4 / WPR;
    const long long ngroups = (a.rows + RPW - 1) / RPW;
    const long long grid = ngroups < kMaxGrid ? ngroups : kMaxGrid;
    hipLaunchKernelGGL((softmax_rows_kernel<ET, WPR, VEC>), dim3((unsigned)grid), dim3(kThreads), 0,
                       (hipStream_t)a.stream, a.a, a.ls, a.p, a.rows, a.cols, a.scale, ngroups);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_et(const SoftmaxArgs& a) {
    const bool vec = a.cols % Elem<ET>::kPerChunk == 0;
    const long long chunks = a.cols / Elem<ET>::kPerChunk;
    // Register rows pay off when p is written (no second read) and for short
    // rows; the statistics alone of longer rows stream faster (measured: more
    // waves in flight with the few registers the streaming kernel needs).
    if (vec && (a.p != nullptr || chunks <= 128)) {
        if (chunks <= 64) return launch_reg<ET, 1>(a);
        if (chunks <= 128) return launch_reg<ET, 2>(a);
        if (chunks <= 256) return launch_reg<ET, 4>(a);
        if (chunks <= 512) return launch_reg<ET, 8>(a);
        if (chunks <= 1024) return launch_reg<ET, 16>(a);
    }
    const bool wide = a.cols > 16384;
    if (wide) return vec ? launch3<ET, 4, true>(a) : launch3<ET, 4, false>(a);
    return vec ? launch3<ET, 1, true>(a) : launch3<ET, 1, false>(a);
}

}  // namespace

hipError_t launch_softmax_rows(const SoftmaxArgs& a) {
    switch (a.dtype) {
        case kF16: return launch_et<kF16>(a);
        case kBF16: return launch_et<kBF16>(a);
        case kF32: return launch_et<kF32>(a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace sdattn
