// twopass.hip -- the partially fused softmax of Sec. 3.2.1 as separate steps:
//
//   1. logits      A = scale Q K^T, written to memory (fp16, bf16 or fp32);
//   2. Eq. 4       (L, S) per row of A -- softmax_rows.hip;
//   3. softmax_pv  O = exp(A - L) / S times V: the element-wise normalisation
//                  fused with the matrix product, reading A once more.
//
// This is the method the paper uses where its FlashAttention kernel does not
// pay off; the A matrix travels through HBM three times (written once, read
// twice).  The single-pass kernel (attn_fwd_kernel.h) never materialises it.
//
// Both kernels use 32x32x16 MFMAs with one query per lane, as the fused
// kernel does.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {


constexpr int kLgQ = 128;   // logits tile: query rows (4 waves x 32)
constexpr int kLgK = 128;   // logits tile: keys
constexpr int kPvQ = 128;   // softmax_pv: query rows per workgroup (4 waves x 32)
constexpr int kPvK = 64;    // softmax_pv: keys per V tile

template <int OT>
constexpr int out_size() { return OT == kF32 ? 4 : 2; }

// ------------------------------------------------------------------ logits

template <int D, int OT>
struct LgGeom {
    static constexpr int DK = (D + 15) / 16;
    static constexpr int kKBytes = kLgK * D * 2;                   // K tile
    static constexpr int kKChunks = (kKBytes + 1023) / 1024;
    static constexpr int kGuard = 16;                              // zeros after the K tile
    static constexpr int kRowBytes = kLgK * out_size<OT>() + 16;   // staging row (padded)
    static constexpr int kStage = kKBytes + kGuard;
    static constexpr int kLdsBytes = kStage + 4 * 32 * kRowBytes;
};

// One workgroup: 128 query rows x 128 keys of one (batch, head); wave w owns
// query rows 32w .. 32w + 31 and all 128 keys (four 32-key sub-tiles of S^T).
template <int ET, int D, int OT>
__global__ __launch_bounds__(256) void logits_kernel(const uint16_t* __restrict__ Q,
                                                     const uint16_t* __restrict__ K, char* __restrict__ A,
                                                     int Lq, int Lk, float scale, int nqt, int nkt,
                                                     int vec_ok) {
    using G = LgGeom<D, OT>;
    constexpr int DK = G::DK;
    constexpr int ES = out_size<OT>();
    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int kt = tile % nkt;
    const int rest = tile / nkt;
    const int qt = rest % nqt;
    const int bh = rest / nqt;
    const int q0 = qt * kLgQ + wave * 32;
    const int k0 = kt * kLgK;

    // K rows k0 .. k0 + 127 (rows past Lk repeat row Lk - 1) into LDS
    const char* Kh = (const char*)(K + (size_t)bh * Lk * D);
#pragma unroll
    for (int i = 0; i < (G::kKChunks + 3) / 4; ++i) {
        const int c = wave + 4 * i;
        if (c < G::kKChunks) {
            const int byte = c * 1024 + lane * 16;
            if (byte < G::kKBytes) {
                const int row = byte / (2 * D);
                const int col = byte - row * (2 * D);
                const size_t goff = (size_t)min(k0 + row, Lk - 1) * (2 * D) + col;
                __builtin_amdgcn_global_load_lds(Kh + goff, (lds_void_t*)(smem + c * 1024), 16, 0, 0);
            }
        }
    }
    if (tid == 0) *(u32x4*)(smem + G::kKBytes) = u32x4{0u, 0u, 0u, 0u};

    // Q^T operand: lane holds query q0 + l32, d = 16s + 8*half .. +7
    const int qrow = q0 + l32;
    u32x4 qreg[DK];
#pragma unroll
    for (int s = 0; s < DK; ++s) {
        const int d0 = 16 * s + 8 * half;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (qrow < Lq && d0 < D) v = *(const u32x4*)(Q + ((size_t)bh * Lq + qrow) * D + d0);
        qreg[s] = v;
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // S^T per 32-key sub-tile, scaled, rounded and staged as rows [query][key]
    char* stage = smem + G::kStage + wave * 32 * G::kRowBytes;
    const int k_off = (l32 * D + 8 * half) * 2;
#pragma unroll
    for (int ks = 0; ks < kLgK / 32; ++ks) {
        f32x16 st;
#pragma unroll
        for (int r = 0; r < 16; ++r) st[r] = 0.0f;
#pragma unroll
        for (int s = 0; s < DK; ++s) {
            const u32x4 a = *(const u32x4*)(smem + k_off + (32 * ks * D + 16 * s) * 2);
            st = mfma32x32x16<ET>(a, qreg[s], st);
        }
        // keys 32ks + 8g + 4*half + (0..3) of row l32
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            char* dst = stage + l32 * G::kRowBytes + (32 * ks + 8 * g + 4 * half) * ES;
            if constexpr (OT == kF32) {
                *(f32x4*)dst = f32x4{st[4 * g] * scale, st[4 * g + 1] * scale, st[4 * g + 2] * scale,
                                     st[4 * g + 3] * scale};
            } else {
                *(u32x2*)dst = u32x2{pack2<OT>(st[4 * g] * scale, st[4 * g + 1] * scale),
                                     pack2<OT>(st[4 * g + 2] * scale, st[4 * g + 3] * scale)};
            }
        }
    }

    // rows of this wave's tile -> A, 16-byte lanes when rows allow it
    const size_t arow0 = (size_t)bh * Lq + q0;
    if (vec_ok && k0 + kLgK <= Lk) {
        constexpr int kLanesPerRow = kLgK * ES / 16;
        constexpr int kRowsPerIter = 64 / kLanesPerRow;
#pragma unroll
        for (int it = 0; it < 32 / kRowsPerIter; ++it) {
            const int r = it * kRowsPerIter + lane / kLanesPerRow;
            const int cb = (lane % kLanesPerRow) * 16;
            if (q0 + r < Lq)
                *(u32x4*)(A + ((arow0 + r) * Lk + k0) * ES + cb) =
                    *(const u32x4*)(stage + r * G::kRowBytes + cb);
        }
    } else {
        const int kn = min(kLgK, Lk - k0);
        for (int r = 0; r < 32; ++r) {
            if (q0 + r >= Lq) break;
            for (int c = lane; c < kn; c += 64) {
                char* dst = A + ((arow0 + r) * Lk + k0 + c) * ES;
                const char* src = stage + r * G::kRowBytes + c * ES;
                if constexpr (ES == 4) *(uint32_t*)dst = *(const uint32_t*)src;
                else *(uint16_t*)dst = *(const uint16_t*)src;
            }
        }
    }
}

// ------------------------------------------------------------- softmax_pv

template <int D>
struct PvGeom {
    static constexpr int DN = (D + 31) / 32;
    static constexpr int kTileBytes = kPvK * D * 2;
    static constexpr int kVPer = (kTileBytes / 16 + 255) / 256;   // 16-byte V pieces per thread
    static constexpr int kLdsBytes = 2 * kTileBytes;               // double-buffered V tiles
};

// One workgroup: 128 query rows of one (batch, head), all keys in 64-key
// tiles; wave w owns rows 32w .. 32w + 31.  Per 16-key step, lane (l32, half)
// takes keys 8*half .. +7 of its row straight from A (16 or 32 bytes), so the
// P^T operand of O^T += V^T P^T needs no shuffle; V^T comes from the row-major
// V tile by transposing LDS reads arranged for that natural key order.
//
// VEC (Lk % 8 == 0): every 8-key piece of A is either wholly inside Lk or
// wholly past it; the pieces of tile t + 2 are loaded while tile t is
// consumed.  Otherwise A is read element by element.
template <int AT, int ET, int D, bool VEC>
__global__ __launch_bounds__(256) void softmax_pv_kernel(const char* __restrict__ A,
                                                         const float* __restrict__ LS,
                                                         const uint16_t* __restrict__ V,
                                                         uint16_t* __restrict__ O, int Lq, int Lk,
                                                         int nqb) {
    using G = PvGeom<D>;
    constexpr int DN = G::DN;
    constexpr int TB = G::kTileBytes;
    constexpr int AS = out_size<AT>();
    constexpr int NV = AS == 4 ? 2 : 1;   // 16-byte pieces per 8 logits
    constexpr int NU = kPvK / 16;         // 16-key steps per tile
    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int bh = tile / nqb;
    const int qb = tile - bh * nqb;
    const int qrow = qb * kPvQ + wave * 32 + l32;
    const bool qvalid = qrow < Lq;
    const size_t row = (size_t)bh * Lq + (qvalid ? qrow : 0);   // rows past Lq read row 0

    const char* Vh = (const char*)(V + (size_t)bh * Lk * D);
    const char* arow = A + row * Lk * AS;
    // weights exp(a - L) 2^8 (the largest 256 rather than 1, so that weights
    // down to 2^-32 of it stay above fp16's smallest subnormal); the factor
    // comes out with 1 / S
    const float cL = LS[2 * row] * kLog2e - 8.0f;
    const float Sinv = (1.0f / 256.0f) / LS[2 * row + 1];
    const int ntiles = (Lk + kPvK - 1) / kPvK;

    // V tile t into registers (rows past Lk are zero), then into LDS buffer b
    u32x4 vreg[G::kVPer];
    auto load_v = [&](int t) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < G::kVPer; ++i) {
            const int byte = (tid + 256 * i) * 16;
            vreg[i] = u32x4{0u, 0u, 0u, 0u};
            if (byte < TB) {
                const int r = byte / (2 * D);
                const int k = t * kPvK + r;
                if (k < Lk) vreg[i] = *(const u32x4*)(Vh + (size_t)k * (2 * D) + (byte - r * 2 * D));
            }
        }
    };
    auto store_v = [&](int b) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < G::kVPer; ++i) {
            const int byte = (tid + 256 * i) * 16;
            if (byte < TB) *(u32x4*)(smem + b * TB + byte) = vreg[i];
        }
    };

    // V^T operand offsets: within each 16-lane group g, lane i points at key
    // 8*(g/2) + i/4 (and +4 for the second read), d = 32n + 16*(g%2) + 4*(i%4).
    int v_off[DN];
    {
        const int g = lane >> 4, i = lane & 15;
        const int krow = 8 * (g >> 1) + (i >> 2);
#pragma unroll
        for (int n = 0; n < DN; ++n) {
            const int ds = 32 * n + 16 * (g & 1) + 4 * (i & 3);
            v_off[n] = (krow * D + (ds < D ? ds : 0)) * 2;   // rows past D of O^T are unused
        }
    }

    // Raw A pieces of one tile for this lane: step u covers keys
    // t*64 + 16u + 8*half .. +7.  Pieces past Lk read the row's first keys
    // (in bounds) and are dropped when converted.
    typedef u32x4 Raw[NU][NV];
    auto fetch = [&](int t, Raw& raw) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int kb = t * kPvK + 16 * u + 8 * half;
            const int ks = kb < Lk ? kb : 0;
#pragma unroll
            for (int v = 0; v < NV; ++v) raw[u][v] = *(const u32x4*)(arow + (size_t)ks * AS + 16 * v);
        }
    };
    // p for keys kb .. kb + 7 from 8 logits a[]: exp2(a log2e - L log2e), 0 past Lk
    auto make_p = [&](const float* a, int kb) __attribute__((always_inline)) -> u32x4 {
        u32x4 pk;
#pragma unroll
        for (int w = 0; w < 4; ++w)
            pk[w] = pack2<ET>(fast_exp2(fmaf(a[2 * w], kLog2e, -cL)),
                              fast_exp2(fmaf(a[2 * w + 1], kLog2e, -cL)));
        return (qvalid && kb < Lk) ? pk : u32x4{0u, 0u, 0u, 0u};
    };
    auto convert = [&](int t, const Raw& raw, u32x4 (&pk)[NU]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            float a[8];
            if constexpr (AS == 4) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    a[e] = __uint_as_float(raw[u][0][e]);
                    a[4 + e] = __uint_as_float(raw[u][1][e]);
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    a[2 * e] = to_float<AT>((uint16_t)(raw[u][0][e] & 0xffffu));
                    a[2 * e + 1] = to_float<AT>((uint16_t)(raw[u][0][e] >> 16));
                }
            }
            pk[u] = make_p(a, t * kPvK + 16 * u + 8 * half);
        }
    };
    auto gather = [&](int t, u32x4 (&pk)[NU]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int kb = t * kPvK + 16 * u + 8 * half;
            float a[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                a[e] = -__builtin_inff();
                if (kb + e < Lk) {
                    if constexpr (AS == 4) a[e] = *(const float*)(arow + (size_t)(kb + e) * 4);
                    else a[e] = to_float<AT>(*(const uint16_t*)(arow + (size_t)(kb + e) * 2));
                }
            }
            pk[u] = make_p(a, kb);
        }
    };

    f32x16 acc[DN];
#pragma unroll
    for (int n = 0; n < DN; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[n][r] = 0.0f;

    auto mfma_tile = [&](int b, const u32x4 (&pk)[NU]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < NU; ++u)
#pragma unroll
            for (int n = 0; n < DN; ++n) {
                const char* vb = smem + b * TB + v_off[n] + 16 * u * D * 2;
                const u32x2 lo = lds_read_tr(vb);
                const u32x2 hi = lds_read_tr(vb + 4 * D * 2);
                acc[n] = mfma32x32x16<ET>(u32x4{lo[0], lo[1], hi[0], hi[1]}, pk[u], acc[n]);
            }
    };

    // Tile t: V(t) sits in buffer t & 1 (written before the barrier), V(t + 1)
    // in registers goes to the other buffer, V(t + 2) is loaded.
    load_v(0);
    store_v(0);
    if (ntiles > 1) load_v(1);
    if constexpr (VEC) {
        Raw raw0, raw1;
        fetch(0, raw0);
        fetch(1 < ntiles ? 1 : 0, raw1);
        auto step = [&](int t, Raw& raw) __attribute__((always_inline)) {
            const int b = t & 1;
            __syncthreads();
            if (t + 1 < ntiles) store_v(b ^ 1);
            if (t + 2 < ntiles) load_v(t + 2);
            u32x4 pk[NU];
            convert(t, raw, pk);
            fetch(t + 2 < ntiles ? t + 2 : 0, raw);
            mfma_tile(b, pk);
        };
        for (int t = 0; t < ntiles; t += 2) {
            step(t, raw0);
            if (t + 1 < ntiles) step(t + 1, raw1);
        }
    } else {
        for (int t = 0; t < ntiles; ++t) {
            const int b = t & 1;
            __syncthreads();
            if (t + 1 < ntiles) store_v(b ^ 1);
            if (t + 2 < ntiles) load_v(t + 2);
            u32x4 pk[NU];
            gather(t, pk);
            mfma_tile(b, pk);
        }
    }

    if (qvalid) {
        uint16_t* orow = O + row * D;
#pragma unroll
        for (int n = 0; n < DN; ++n)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int d0 = 32 * n + 8 * g + 4 * half;
                if (32 * n + 8 * g < D) {   // D % 8 == 0: then d0 + 3 < D for both halves
                    u32x2 w;
                    w[0] = pack2<ET>(acc[n][4 * g + 0] * Sinv, acc[n][4 * g + 1] * Sinv);
                    w[1] = pack2<ET>(acc[n][4 * g + 2] * Sinv, acc[n][4 * g + 3] * Sinv);
                    *(u32x2*)(orow + d0) = w;
                }
            }
    }
}

// --------------------------------------------------------------- launchers

template <int ET, int OT, int D>
hipError_t launch_logits_d(const LogitsArgs& a) {
    using G = LgGeom<D, OT>;
    static_assert(G::kLdsBytes <= 160 * 1024, "LDS");
    const int nqt = (a.Lq + kLgQ - 1) / kLgQ;
    const int nkt = (a.Lk + kLgK - 1) / kLgK;
    const long long nblk = (long long)a.B * a.H * nqt * nkt;
    const int vec_ok = ((long long)a.Lk * out_size<OT>()) % 16 == 0;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&logits_kernel<ET, D, OT>),
        hipFuncAttributeMaxDynamicSharedMemorySize, G::kLdsBytes);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL((logits_kernel<ET, D, OT>), dim3((unsigned)nblk), dim3(256), G::kLdsBytes,
                       (hipStream_t)a.stream, (const uint16_t*)a.q, (const uint16_t*)a.k, (char*)a.a,
                       a.Lq, a.Lk, a.scale, nqt, nkt, vec_ok);
    return hipGetLastError();
}

template <int AT, int ET, int D, bool VEC>
hipError_t launch_pv_dv(const SoftmaxPvArgs& a) {
    using G = PvGeom<D>;
    const int nqb = (a.Lq + kPvQ - 1) / kPvQ;
    const long long nblk = (long long)a.B * a.H * nqb;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&softmax_pv_kernel<AT, ET, D, VEC>),
        hipFuncAttributeMaxDynamicSharedMemorySize, G::kLdsBytes);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL((softmax_pv_kernel<AT, ET, D, VEC>), dim3((unsigned)nblk), dim3(256),
                       G::kLdsBytes, (hipStream_t)a.stream, (const char*)a.a, a.ls,
                       (const uint16_t*)a.v, (uint16_t*)a.out, a.Lq, a.Lk, nqb);
    return hipGetLastError();
}

template <int AT, int ET, int D>
hipError_t launch_pv_d(const SoftmaxPvArgs& a) {
    return a.Lk % 8 == 0 ? launch_pv_dv<AT, ET, D, true>(a) : launch_pv_dv<AT, ET, D, false>(a);
}

template <int ET, int OT, int... Ds>
hipError_t dispatch_logits(const LogitsArgs& a, std::integer_sequence<int, Ds...>) {
    hipError_t r = hipErrorInvalidValue;
    bool hit = ((a.D == 8 * (Ds + 1) ? (r = launch_logits_d<ET, OT, 8 * (Ds + 1)>(a), true) : false) || ...);
    return hit ? r : hipErrorInvalidValue;
}

template <int AT, int ET, int... Ds>
hipError_t dispatch_pv(const SoftmaxPvArgs& a, std::integer_sequence<int, Ds...>) {
    hipError_t r = hipErrorInvalidValue;
    bool hit = ((a.D == 8 * (Ds + 1) ? (r = launch_pv_d<AT, ET, 8 * (Ds + 1)>(a), true) : false) || ...);
    return hit ? r : hipErrorInvalidValue;
}

}  // namespace

long long logits_grid(int B, int H, int Lq, int Lk) {
    return (long long)B * H * ((Lq + kLgQ - 1) / kLgQ) * ((Lk + kLgK - 1) / kLgK);
}

hipError_t launch_logits(const LogitsArgs& a) {
    using Seq = std::make_integer_sequence<int, 32>;   // D = 8, 16, ..., 256
    if (a.dtype == kF16) {
        if (a.a_dtype == kF16) return dispatch_logits<kF16, kF16>(a, Seq{});
        if (a.a_dtype == kBF16) return dispatch_logits<kF16, kBF16>(a, Seq{});
        return dispatch_logits<kF16, kF32>(a, Seq{});
    }
    if (a.a_dtype == kF16) return dispatch_logits<kBF16, kF16>(a, Seq{});
    if (a.a_dtype == kBF16) return dispatch_logits<kBF16, kBF16>(a, Seq{});
    return dispatch_logits<kBF16, kF32>(a, Seq{});
}

hipError_t launch_softmax_pv(const SoftmaxPvArgs& a) {
    using Seq = std::make_integer_sequence<int, 32>;
    if (a.dtype == kF16) {
        if (a.a_dtype == kF16) return dispatch_pv<kF16, kF16>(a, Seq{});
        if (a.a_dtype == kBF16) return dispatch_pv<kBF16, kF16>(a, Seq{});
        return dispatch_pv<kF32, kF16>(a, Seq{});
    }
    if (a.a_dtype == kF16) return dispatch_pv<kF16, kBF16>(a, Seq{});
    if (a.a_dtype == kBF16) return dispatch_pv<kBF16, kBF16>(a, Seq{});
    return dispatch_pv<kF32, kBF16>(a, Seq{});
}

}  // namespace sdattn
