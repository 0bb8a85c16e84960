// attn_fwd.hip -- single-pass attention forward (Eq. 3) for gfx950, with the
// K and V tiles streamed into LDS by direct global->LDS copies.
//
// One workgroup = 4 waves = 128 query rows of one (batch, head); each wave
// owns 32 rows.  Keys and values move through LDS in tiles of 64 keys; while
// tiles are consumed, later ones are copied straight from global memory into
// free buffers (global_load_lds, 16 bytes per lane, no
// registers involved).  Both tiles keep the row-major [key][d] layout of
// global memory; a ring of four buffers lets the copy run two tiles ahead.
// Per tile and wave:
//
//   S^T = K Q^T      32x32x16 MFMA.  A = K rows read from LDS (16 bytes per
//                    lane), B = Q^T held in registers for the whole kernel.
//                    The accumulator puts one query per lane (lane % 32) and 16
//                    of a sub-tile's 32 keys in that lane, so the row maximum
//                    needs a single exchange between lane halves.
//   p = 2^(c s - m)  c = |scale| log2(e); the running maximum m moves (with
//                    the matching rescale of O and l) only when a tile's
//                    maximum exceeds it by more than 8, so p <= 256.
//   O^T += V^T P^T   32x32x16 MFMA.  B = P straight from the S^T registers;
//                    A = V^T, produced from the row-major V tile by the
//                    transposing LDS read ds_read_b64_tr_b16: 16 lanes each
//                    point at 4 consecutive d of one key, and every lane gets
//                    4 consecutive keys of one d.
//   l                row sum of the rounded p.  When D is not a multiple of 32,
//                    the lanes whose d lies past D read a constant block
//                    instead of V: a one at d = D and zeros beyond, so the P V
//                    product also yields l in row D of O^T.  Otherwise the
//                    packed p pairs are summed with v_dot2 against (1, 1).
//
// This is the block-wise ("multi-stage") reduction of Sec. 3.2.1 -- a tile's
// maximum and exponential sum merged into the running pair -- fused with the
// element-wise normalisation and the product with V, so the N x M matrix A
// never leaves the chip (the IO-aware tiling of FlashAttention, Sec. 3.2.2).
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kBQ = kWaves * 32;   // query rows per workgroup
constexpr int kKB = 64;            // keys per LDS tile
constexpr float kRescaleSlack = 8.0f;
constexpr int kMaxLds = 160 * 1024;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

template <int D>
struct Geom {
    static constexpr int DK = (D + 15) / 16;                  // 16-deep k steps of Q K^T
    static constexpr int DN = (D + 31) / 32;                  // 32-row d tiles of O^T
    static constexpr bool kOnes = (D % 32) != 0;              // padding rows carry the row sum
    static constexpr int kTileBytes = kKB * D * 2;            // one K or V tile
    static constexpr int kChunks = kTileBytes / 1024;         // 1 KiB wave copies per tile
    static constexpr int kBufBytes = kTileBytes * (kOnes ? 3 : 2);   // K, V (, constant block)
    static constexpr int kLdsBytes = 4 * kBufBytes;   // a ring of four tile buffers
    static constexpr bool kFits = D >= 32 && D % 8 == 0 && kLdsBytes <= kMaxLds;
};

// Logical tile for workgroup `bid`.  Workgroups are dealt round-robin over the
// 8 XCDs; give every XCD a contiguous run of logical tiles so that the tiles
// of one (batch, head) -- which read the same K and V -- share one L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    const int per = nblk / 8, rem = nblk % 8;
    const int xcd = bid % 8, slot = bid / 8;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

__device__ __forceinline__ u32x2 lds_read_tr(const char* p) {
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
    return __builtin_bit_cast(u32x2, v);
}

template <int ET, int D>
__global__ __launch_bounds__(kThreads) void attn_fwd_lds_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    uint16_t* __restrict__ O, float* __restrict__ LS, int Lq, int Lk, float scale_abs, float c,
    int neg, int nqb) {
    using G = Geom<D>;
    constexpr int DK = G::DK;
    constexpr int DN = G::DN;
    constexpr int TB = G::kTileBytes;

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

    // Constant blocks (one per buffer): a one in column 0 of every row, zeros
    // elsewhere.  Lanes whose d lies at or past D read these instead of V.
    if constexpr (G::kOnes) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            uint16_t* cb = (uint16_t*)(smem + b * G::kBufBytes + 2 * TB);
            for (int i = tid; i < kKB * D; i += kThreads)
                cb[i] = (i % D == 0) ? from_float<ET>(1.0f) : (uint16_t)0;
        }
    }

    // Copy key tile [kbase, kbase + 64) of K and V into buffer b.  Wave w
    // issues the 1 KiB pieces w, w + 4, ...; in a tail tile (TAIL), rows past
    // Lk repeat row Lk - 1 (finite data; their weights are forced to zero).
    auto issue_tile = [&](auto tail_c, int kbase, int b) __attribute__((always_inline)) {
        constexpr bool TAIL = decltype(tail_c)::value;
#pragma unroll
        for (int i = 0; i < (2 * G::kChunks + kWaves - 1) / kWaves; ++i) {
            const int cidx = wave + kWaves * i;
            if (cidx < 2 * G::kChunks) {
                const bool isv = cidx >= G::kChunks;
                const int cc = isv ? cidx - G::kChunks : cidx;
                const char* src = isv ? Vh : Kh;
                const int byte = cc * 1024 + lane * 16;
                size_t goff;
                if constexpr (TAIL) {
                    const int row = byte / (2 * D);
                    const int col = byte - row * (2 * D);
                    const int grow = min(kbase + row, Lk - 1);
                    goff = (size_t)grow * (2 * D) + col;
                } else {
                    goff = (size_t)kbase * (2 * D) + byte;
                }
                char* dst = smem + b * G::kBufBytes + (isv ? TB : 0) + cc * 1024;
                __builtin_amdgcn_global_load_lds(src + goff, (lds_void_t*)dst, 16, 0, 0);
            }
        }
    };
    std::integral_constant<bool, false> full_c;
    std::integral_constant<bool, true> tail_c;
    const int nfull = Lk / kKB;
    const int ntiles = (Lk + kKB - 1) / kKB;
    // copy tile t (full or tail) into buffer t % 4, if it exists
    auto issue = [&](int t) __attribute__((always_inline)) {
        if (t < nfull) issue_tile(full_c, t * kKB, t & 3);
        else if (t < ntiles) issue_tile(tail_c, t * kKB, t & 3);
    };

    // Q^T operand: lane holds query q0 + l32, d = 16s + 8*half .. +7 for each s.
    const int qrow = q0 + l32;
    u32x4 qreg[DK];
#pragma unroll
    for (int s = 0; s < DK; ++s) {
        const int d0 = 16 * s + 8 * half;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (qrow < Lq && d0 < D) v = *(const u32x4*)(Q + ((size_t)bh * Lq + qrow) * D + d0);
        if (neg) v ^= 0x80008000u;   // fold a negative scale into Q (exact)
        qreg[s] = v;
    }

    // Per-lane LDS byte offsets inside a buffer.
    // K rows: lane reads key row l32 at d = 8*half (+16 s, +32 t rows).
    const int k_off = (l32 * D + 8 * half) * 2;
    // V^T via transposing reads: 16-lane group g = lane / 16 covers keys
    // 4*(g/2) .. +3 and d = 32n + 16*(g%2) .. +15; its lane i points at key
    // 4*(g/2) + i/4, d = 32n + 16*(g%2) + 4*(i%4) .. +3.
    int v_off[DN];
    {
        const int g = lane >> 4, i = lane & 15;
        const int krow = 4 * (g >> 1) + (i >> 2);
#pragma unroll
        for (int n = 0; n < DN; ++n) {
            const int ds = 32 * n + 16 * (g & 1) + 4 * (i & 3);
            v_off[n] = ds < D ? TB + (krow * D + ds) * 2 : 2 * TB + (krow * D + ds - D) * 2;
        }
    }

    f32x16 acc[DN];
#pragma unroll
    for (int n = 0; n < DN; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[n][r] = 0.0f;
    float m_run = -__builtin_inff();   // running max used in the exponent (log2 units)
    float s_max = -__builtin_inff();   // true running max of the raw scores
    float l_part = 0.0f;               // this lane's part of the row sum (v_dot2 path)

    struct Scores { f32x16 v[2]; };    // S^T of a tile's two 32-key sub-tiles
    struct Probs { u32x4 v[2][2]; };   // its rounded p as four P^T operands

    // S^T = K Q^T for the tile in buffer BUF
    auto qk = [&](auto buf_c) __attribute__((always_inline)) {
        constexpr int BUF = decltype(buf_c)::value;
        const char* base = smem + BUF * G::kBufBytes;
        Scores st;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) st.v[t][r] = 0.0f;
#pragma unroll
            for (int s = 0; s < DK; ++s) {
                const u32x4 a = *(const u32x4*)(base + k_off + (32 * t * D + 16 * s) * 2);
                st.v[t] = mfma32x32x16<ET>(a, qreg[s], st.v[t]);
            }
        }
        return st;
    };

    // O^T += V^T P^T with V from buffer BUF; keys of operand slot e are
    // 32t + 16u + 8*(e/4) + 4*half + e%4
    auto pv = [&](auto buf_c, const Probs& pk) __attribute__((always_inline)) {
        constexpr int BUF = decltype(buf_c)::value;
        const char* base = smem + BUF * G::kBufBytes;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int n = 0; n < DN; ++n) {
                    const char* vb = base + v_off[n];
                    const u32x2 lo = lds_read_tr(vb + (32 * t + 16 * u) * D * 2);
                    const u32x2 hi = lds_read_tr(vb + (32 * t + 16 * u + 8) * D * 2);
                    const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                    acc[n] = mfma32x32x16<ET>(a, pk.v[t][u], acc[n]);
                }
    };

    // Softmax step of a tile (keys kbase ..): merge its row maximum into the
    // running one, p = 2^(c s - m) rounded to the input type.  The decision
    // to move m is wave-uniform and taken without a branch; the matching
    // rescale of O (alpha != 1) is left to the caller, after the MFMAs that
    // still accumulate the previous tile into O.
    auto softmax = [&](auto tail_c, Scores st, int kbase, float& alpha, bool& moved)
                       __attribute__((always_inline)) {
        constexpr bool TAIL = decltype(tail_c)::value;
        if constexpr (TAIL) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kbase + 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (key >= Lk) st.v[t][r] = -__builtin_inff();
                }
        }
        float mloc = st.v[0][0];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, st.v[t][r]);
        mloc = half_max(mloc);
        s_max = fmaxf(s_max, mloc);
        const float mb = mloc * c;
        moved = __any(mb > m_run + kRescaleSlack);
        const float m_new = moved ? fmaxf(m_run, mb) : m_run;
        alpha = moved ? fast_exp2(m_run - m_new) : 1.0f;
        m_run = m_new;
        const float negm = -m_run;
        Probs pk;
        if constexpr (!G::kOnes) l_part *= alpha;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            float p[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) p[r] = fast_exp2(fmaf(st.v[t][r], c, negm));
            if constexpr (TAIL) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kbase + 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (key >= Lk) p[r] = 0.0f;
                }
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w) pk.v[t][u][w] = pack2<ET>(p[8 * u + 2 * w], p[8 * u + 2 * w + 1]);
            if constexpr (!G::kOnes) {
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int w = 0; w < 4; ++w) l_part = add_pair<ET>(pk.v[t][u][w], l_part);
            }
        }
        return pk;
    };

    auto rescale = [&](float alpha) __attribute__((always_inline)) {
#pragma unroll
        for (int n = 0; n < DN; ++n)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[n][r] *= alpha;
    };

    // Interleave the step's matrix-core work (P V of the previous tile, then
    // S of the next) with the softmax of the current tile: one MFMA, a few
    // LDS reads for the next MFMA, then a run of vector instructions.
    auto interleave = [&]() __attribute__((always_inline)) {
        constexpr int kPV = 4 * DN, kQK = 2 * DK;
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * kPV + kQK, 0);   // every LDS read first
#pragma unroll
        for (int i = 0; i < kPV; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);   // VALU
        }
#pragma unroll
        for (int i = 0; i < kQK; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
        }
    };

    // Software pipeline over tiles, four LDS buffers (tile t lives in buffer
    // t % 4).  A middle step j (tile j full, tile j+1 present):
    //   - starts copying tile j+2,
    //   - multiplies the previous tile's P by V (tile j-1),
    //   - does the softmax of tile j (its scores are already in registers),
    //   - computes the scores of tile j+1,
    // so the matrix cores work on tiles j-1 and j+1 while the vector ALU works
    // on tile j.  One barrier per step publishes tile j+2 and frees buffer
    // (j-1) % 4 for the copy issued at step j+1.
    Scores S;      // scores of the tile being softmaxed
    Probs P;       // probabilities of the tile before it

    auto mid_step = [&](auto bj_c, auto has_prev_c, int j) __attribute__((always_inline)) {
        constexpr int BJ = decltype(bj_c)::value;   // j % 4
        constexpr bool PREV = decltype(has_prev_c)::value;
        std::integral_constant<int, (BJ + 1) % 4> bn_c;
        std::integral_constant<int, (BJ + 3) % 4> bp_c;
        issue(j + 2);
        if constexpr (PREV) pv(bp_c, P);
        float alpha;
        bool moved;
        const Probs pc = softmax(full_c, S, j * kKB, alpha, moved);
        S = qk(bn_c);
        interleave();
        if (moved) rescale(alpha);
        P = pc;
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    };

    // The last tile (j = ntiles - 1): previous P V, masked softmax, own P V.
    auto last_step = [&](auto bj_c, auto has_prev_c, int j) __attribute__((always_inline)) {
        constexpr int BJ = decltype(bj_c)::value;
        constexpr bool PREV = decltype(has_prev_c)::value;
        std::integral_constant<int, (BJ + 3) % 4> bp_c;
        if constexpr (PREV) pv(bp_c, P);
        float alpha;
        bool moved;
        const Probs pc = (j < nfull) ? softmax(full_c, S, j * kKB, alpha, moved)
                                     : softmax(tail_c, S, j * kKB, alpha, moved);
        if (moved) rescale(alpha);
        pv(bj_c, pc);
    };

    std::integral_constant<int, 0> c0;
    std::integral_constant<int, 1> c1;
    std::integral_constant<int, 2> c2;
    std::integral_constant<int, 3> c3;
    std::integral_constant<bool, false> noprev_c;
    std::integral_constant<bool, true> prev_c;

    issue(0);
    issue(1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    S = qk(c0);
    if (ntiles == 1) {
        last_step(c0, noprev_c, 0);
    } else {
        mid_step(c0, noprev_c, 0);
        int j = 1;
        for (; j + 4 < ntiles; j += 4) {
            mid_step(c1, prev_c, j);
            mid_step(c2, prev_c, j + 1);
            mid_step(c3, prev_c, j + 2);
            mid_step(c0, prev_c, j + 3);
        }
        if (j + 1 < ntiles) {
            mid_step(c1, prev_c, j++);
            if (j + 1 < ntiles) {
                mid_step(c2, prev_c, j++);
                if (j + 1 < ntiles) mid_step(c3, prev_c, j++);
            }
        }
        switch (j & 3) {
            case 0: last_step(c0, prev_c, j); break;
            case 1: last_step(c1, prev_c, j); break;
            case 2: last_step(c2, prev_c, j); break;
            default: last_step(c3, prev_c, j); break;
        }
    }

    // ---- epilogue: l, O / l, store
    float l;
    if constexpr (G::kOnes) {
        constexpr int dd = D % 32;               // position of the ones row in its d tile
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
            // Eq. 4 in natural units: L = max_j scale q.k, S = sum_j exp(scale q.k - L)
            float* o2 = LS + ((size_t)bh * Lq + qrow) * 2;
            o2[0] = s_max * scale_abs;
            o2[1] = l * fast_exp2(m_run - s_max * c);
        }
    }
}

template <int ET, int D>
hipError_t launch_d(const AttnArgs& a) {
    using G = Geom<D>;
    if constexpr (!G::kFits) {
        return launch_attn_fwd_generic(a);
    } else {
        const int nqb = (a.Lq + kBQ - 1) / kBQ;
        const long long nblk = (long long)a.B * a.H * nqb;
        const float scale_abs = a.scale < 0 ? -a.scale : a.scale;
        const float c = scale_abs * kLog2e;
        static const hipError_t attr = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&attn_fwd_lds_kernel<ET, D>),
            hipFuncAttributeMaxDynamicSharedMemorySize, G::kLdsBytes);
        if (attr != hipSuccess) return attr;
        hipLaunchKernelGGL((attn_fwd_lds_kernel<ET, D>), dim3((unsigned)nblk), dim3(kThreads),
                           G::kLdsBytes, (hipStream_t)a.stream, (const uint16_t*)a.q,
                           (const uint16_t*)a.k, (const uint16_t*)a.v, (uint16_t*)a.out, a.ls,
                           a.Lq, a.Lk, scale_abs, c, a.scale < 0 ? 1 : 0, nqb);
        return hipGetLastError();
    }
}

template <int ET, int... Ds>
hipError_t dispatch_d(const AttnArgs& a, std::integer_sequence<int, Ds...>) {
    hipError_t r = hipErrorInvalidValue;
    bool hit = ((a.D == 8 * (Ds + 1) ? (r = launch_d<ET, 8 * (Ds + 1)>(a), true) : false) || ...);
    return hit ? r : hipErrorInvalidValue;
}

}  // namespace

long long attn_fwd_grid(int B, int H, int Lq) {
    return (long long)B * H * ((Lq + kBQ - 1) / kBQ);
}

hipError_t launch_attn_fwd(const AttnArgs& a) {
    if (attn_fwd_short_supported(a.D, a.Lk)) return launch_attn_fwd_short(a);
    if (a.D < 32) return launch_attn_fwd_generic(a);
    using Seq = std::make_integer_sequence<int, 32>;   // D = 8, 16, ..., 256
    return a.dtype == kF16 ? dispatch_d<kF16>(a, Seq{}) : dispatch_d<kBF16>(a, Seq{});
}

}  // namespace sdattn
