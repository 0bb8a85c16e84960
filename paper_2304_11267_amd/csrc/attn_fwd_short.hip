// attn_fwd_short.hip -- attention forward (Eq. 3) for short key sequences
// (Lk <= 128), the cross-attention over SD's 77-token text context.
//
// Every key and value of a (batch, head) fits in LDS at once, so the kernel
// reads them a single time, computes the exact row maximum over all keys (no
// running maximum, no rescale of O) and then p and P V -- Eq. 4's reduction
// and the element-wise step in one pass over registers.
//
// The work is bound by streaming Q in and O out of HBM, so both move as whole
// contiguous blocks: a wave's 32 query rows are one run of 32*D*2 bytes, which
// the wave copies into LDS with 1 KiB direct global->LDS loads and reads back
// in MFMA operand order; the normalised O tile goes the other way, written to
// the same LDS region in row-major order and stored with 16-byte lanes.
//
// Keys are processed in NS = ceil(Lk / 32) sub-tiles of 32.  Key rows past
// Lk repeat row Lk - 1, so their scores never exceed the true maximum and no
// mask is needed for it.  Their value rows, and their entries in the row of
// ones, are zero, so their p adds nothing to O or to the row sum; only when D
// is a multiple of 32 (the row sum then comes from the p registers) does the
// last sub-tile mask p past Lk.  The P V product skips a final 16-key step
// that lies wholly past Lk.  A negative scale negates K once in LDS.
//
// A workgroup holds W = 4 waves (one 32-row strip each) and loads K and V
// once for all of them.
//
// Operand layouts are those of the long-sequence kernel: S^T = K Q^T and
// O^T = V^T P^T on 32x32x16 MFMAs with one query per lane, V^T produced by
// ds_read_b64_tr_b16 from row-major V, and the row sum taken from a row of
// ones at d = D when D is not a multiple of 32.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

template <int D, int NS, int W>
struct ShortGeom {
    static constexpr int DK = (D + 15) / 16;
    static constexpr int DN = (D + 31) / 32;
    static constexpr bool kOnes = (D % 32) != 0;
    static constexpr int kRows = 32 * NS;                        // key rows held in LDS
    static constexpr int kBlockBytes = kRows * D * 2;            // K, V or the constant block
    static constexpr int kChunks = (kBlockBytes + 1023) / 1024;  // 1 KiB wave copies per block
    static constexpr int kStripBytes = 32 * D * 2;               // one wave's Q (then O) rows
    static constexpr int kStripChunks = (kStripBytes + 1023) / 1024;
    static constexpr int kV = kBlockBytes;
    static constexpr int kC = 2 * kBlockBytes;
    static constexpr int kQ = (kOnes ? 3 : 2) * kBlockBytes;
    static constexpr int kLdsBytes = kQ + W * kStripBytes;
    static constexpr bool kFits = kLdsBytes <= 160 * 1024;
    static_assert(kBlockBytes % 16 == 0 && kStripBytes % 16 == 0, "16-byte LDS chunks");
};

// Arguments used first come first, so they fit in the preloaded kernel-argument
// registers.
template <int ET, int D, int NS, int W>
__global__ __launch_bounds__(W * 64) void attn_fwd_short_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    uint16_t* __restrict__ O, int Lq, int Lk, float c, int nqb, int nblk, int neg,
    float* __restrict__ LS, float scale_abs, int oh) {
    using G = ShortGeom<D, NS, W>;
    constexpr int kThreads = W * 64;
    constexpr int DK = G::DK;
    constexpr int DN = G::DN;
    constexpr int BB = G::kBlockBytes;

    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int tile = xcd_remap(blockIdx.x, nblk);
    const int bh = tile / nqb;
    const int qb = tile - bh * nqb;
    const int q0 = qb * (32 * W) + wave * 32;
    // bytes of this wave's 32-row strip that lie inside Q / O (<= 0: none)
    const int strip_bytes = min(32, Lq - q0) * (2 * D);
    char* stage = smem + G::kQ + wave * G::kStripBytes;

    const char* Kh = (const char*)(K + (size_t)bh * Lk * D);
    const char* Vh = (const char*)(V + (size_t)bh * Lk * D);

    // K and V rows 0 .. 32*NS - 1, 1 KiB per wave copy of the contiguous rows
    // below Lk; past them K repeats row Lk - 1 and V is zero.
    const int kv_bytes = Lk * (2 * D);
#pragma unroll
    for (int i = 0; i < (2 * G::kChunks + W - 1) / W; ++i) {
        const int cidx = wave + W * i;
        if (cidx < 2 * G::kChunks) {
            const bool isv = cidx >= G::kChunks;
            const int cc = isv ? cidx - G::kChunks : cidx;
            const int byte = cc * 1024 + lane * 16;
            const char* src = isv ? Vh : Kh;
            char* dst = smem + (isv ? G::kV : 0) + cc * 1024;
            if (cc * 1024 + 1024 <= kv_bytes) {
                __builtin_amdgcn_global_load_lds(src + byte, (lds_void_t*)dst, 16, 0, 0);
            } else if (byte < BB) {
                if (byte < kv_bytes) {
                    __builtin_amdgcn_global_load_lds(src + byte, (lds_void_t*)dst, 16, 0, 0);
                } else if (!isv) {
                    const int col = (byte - kv_bytes) % (2 * D);
                    __builtin_amdgcn_global_load_lds(src + (kv_bytes - 2 * D) + col, (lds_void_t*)dst,
                                                     16, 0, 0);
                } else {
                    *(u32x4*)(dst + lane * 16) = u32x4{0u, 0u, 0u, 0u};
                }
            }
        }
    }

    // This wave's Q rows, one contiguous run.
    {
        const char* qs = (const char*)(Q + ((size_t)bh * Lq + q0) * D);
#pragma unroll
        for (int i = 0; i < G::kStripChunks; ++i) {
            const int byte = i * 1024 + lane * 16;
            if (byte < strip_bytes)
                __builtin_amdgcn_global_load_lds(qs + byte, (lds_void_t*)(stage + i * 1024), 16, 0, 0);
        }
    }

    // Row-sum column: V^T row D is read from a block with V's row stride whose
    // first four columns hold (1, 0, 0, 0) for key rows below Lk and zeros past
    // it; only those four columns are ever read.
    if constexpr (G::kOnes) {
        for (int r = tid; r < G::kRows; r += kThreads) {
            u32x2 w = {r < Lk ? (uint32_t)from_float<ET>(1.0f) : 0u, 0u};
            *(u32x2*)(smem + G::kC + r * (2 * D)) = w;
        }
    }

    const int k_off = (l32 * D + 8 * half) * 2;
    int v_off[DN];
    {
        const int g = lane >> 4, i = lane & 15;
        const int krow = 4 * (g >> 1) + (i >> 2);
#pragma unroll
        for (int n = 0; n < DN; ++n) {
            // rows past D + 3 of O^T are never used: those lanes read V
            const int ds = 32 * n + 16 * (g & 1) + 4 * (i & 3);
            v_off[n] = ds == D ? G::kC + krow * D * 2
                               : G::kV + (krow * D + (ds < D ? ds : ds - 32)) * 2;
        }
    }

    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    if (neg) {   // scale < 0: softmax(scale * q.k) = softmax(|scale| * q.(-k))
        for (int i = tid; i < BB / 16; i += kThreads) *(u32x4*)(smem + i * 16) ^= 0x80008000u;
        __syncthreads();
    }

    // Q^T operand: lane holds query q0 + l32, d = 16s + 8*half .. +7 (zero past
    // D).  Rows past Lq hold stale LDS data; they only reach their own lanes'
    // columns of S^T and O^T, which are never stored.
    const bool qvalid = q0 + l32 < Lq;
    u32x4 qreg[DK];
#pragma unroll
    for (int s = 0; s < DK; ++s) {
        const int d0 = 16 * s + 8 * half;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (d0 < D) v = *(const u32x4*)(stage + (l32 * D + d0) * 2);
        qreg[s] = v;
    }

    // S^T for every 32-key sub-tile
    f32x16 st[NS];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
#pragma unroll
        for (int r = 0; r < 16; ++r) st[t][r] = 0.0f;
#pragma unroll
        for (int s = 0; s < DK; ++s) {
            const u32x4 a = *(const u32x4*)(smem + k_off + (32 * t * D + 16 * s) * 2);
            st[t] = mfma32x32x16<ET>(a, qreg[s], st[t]);
        }
    }

    // exact row maximum: padded key rows repeat key Lk - 1
    float mloc = st[0][0];
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, st[t][r]);
    const float s_max = half_max(mloc);
    // weights 2^(c s - c s_max + 8): the largest 256 rather than 1, so that
    // weights down to 2^-32 of it stay above fp16's smallest subnormal (the
    // factor cancels in O / l and is taken out of S below)
    const float negm = 8.0f - s_max * c;

    f32x16 acc[DN];
#pragma unroll
    for (int n = 0; n < DN; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[n][r] = 0.0f;
    float l_part = 0.0f;

#pragma unroll
    for (int t = 0; t < NS; ++t) {
        u32x4 pk[2];
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            p[r] = fast_exp2(fmaf(st[t][r], c, negm));
            if (!G::kOnes && t == NS - 1) {
                const int key = 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                if (key >= Lk) p[r] = 0.0f;
            }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int w = 0; w < 4; ++w) pk[u][w] = pack2<ET>(p[8 * u + 2 * w], p[8 * u + 2 * w + 1]);
        if constexpr (!G::kOnes) {
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w) l_part = add_pair<ET>(pk[u][w], l_part);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (t == NS - 1 && u == 1 && 32 * t + 16 >= Lk) break;
#pragma unroll
            for (int n = 0; n < DN; ++n) {
                const char* vb = smem + v_off[n] + (32 * t + 16 * u) * D * 2;
                const u32x2 lo = lds_read_tr(vb);
                const u32x2 hi = lds_read_tr(vb + 8 * D * 2);
                const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                acc[n] = mfma32x32x16<ET>(a, pk[u], acc[n]);
            }
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

    // O tile -> LDS (row-major, over this wave's Q rows) -> contiguous 16-byte stores.
#pragma unroll
    for (int n = 0; n < DN; ++n)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int d0 = 32 * n + 8 * g + 4 * half;
            if (32 * n + 8 * g < D) {   // D % 8 == 0: then d0 + 3 < D for both halves
                u32x2 w;
                w[0] = pack2<ET>(acc[n][4 * g + 0] * inv, acc[n][4 * g + 1] * inv);
                w[1] = pack2<ET>(acc[n][4 * g + 2] * inv, acc[n][4 * g + 3] * inv);
                *(u32x2*)(stage + (l32 * D + d0) * 2) = w;
            }
        }
    {
        if (oh == 0) {   // the strip's rows are contiguous in O
            char* os = (char*)(O + ((size_t)bh * Lq + q0) * D);
#pragma unroll
            for (int i = 0; i < G::kStripChunks; ++i) {
                const int byte = i * 1024 + lane * 16;
                if (byte < strip_bytes) *(u32x4*)(os + byte) = *(const u32x4*)(stage + byte);
            }
        } else {         // row r of the strip is token q0 + r's slice of channels h*D .. h*D + D - 1
            uint16_t* ob = out_base(O, bh, Lq, D, oh) + (size_t)q0 * out_stride(D, oh);
#pragma unroll
            for (int i = 0; i < G::kStripChunks; ++i) {
                const int byte = i * 1024 + lane * 16;
                if (byte < strip_bytes) {
                    const int r = byte / (2 * D), col = byte - r * (2 * D);
                    *(u32x4*)((char*)(ob + (size_t)r * out_stride(D, oh)) + col) =
                        *(const u32x4*)(stage + byte);
                }
            }
        }
    }
    if (LS && half == 0 && qvalid) {
        float* o2 = LS + ((size_t)bh * Lq + q0 + l32) * 2;
        o2[0] = s_max * scale_abs;
        o2[1] = l * (1.0f / 256.0f);
    }
}

template <int ET, int D, int NS, int W>
hipError_t launch_short_dnw(const AttnArgs& a) {
    using G = ShortGeom<D, NS, W>;
    static_assert(G::kFits, "LDS");
    const int nqb = (a.Lq + 32 * W - 1) / (32 * W);
    const long long nblk = (long long)a.B * a.H * nqb;
    const float scale_abs = a.scale < 0 ? -a.scale : a.scale;
    const float c = scale_abs * kLog2e;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&attn_fwd_short_kernel<ET, D, NS, W>),
        hipFuncAttributeMaxDynamicSharedMemorySize, G::kLdsBytes);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL((attn_fwd_short_kernel<ET, D, NS, W>), dim3((unsigned)nblk), dim3(W * 64),
                       G::kLdsBytes, (hipStream_t)a.stream, (const uint16_t*)a.q,
                       (const uint16_t*)a.k, (const uint16_t*)a.v, (uint16_t*)a.out, a.Lq, a.Lk, c,
                       nqb, (int)nblk, a.scale < 0 ? 1 : 0, a.ls, scale_abs, a.o_rows ? a.H : 0);
    return hipGetLastError();
}

// Four waves per workgroup: at the 64x64 level (2048 strips) this makes two
// workgroups per CU with their own barriers, which measured faster with cold
// inputs than one workgroup of eight (5.24 vs 5.47 us; two waves: 5.77).
template <int ET, int D, int NS>
hipError_t launch_short_dn(const AttnArgs& a) {
    return launch_short_dnw<ET, D, NS, 4>(a);
}

template <int ET, int D>
hipError_t launch_short_d(const AttnArgs& a) {
    switch ((a.Lk + 31) / 32) {
        case 1: return launch_short_dn<ET, D, 1>(a);
        case 2: return launch_short_dn<ET, D, 2>(a);
        case 3: return launch_short_dn<ET, D, 3>(a);
        default: return launch_short_dn<ET, D, 4>(a);
    }
}

template <int ET, int... Ds>
hipError_t dispatch_short(const AttnArgs& a, std::integer_sequence<int, Ds...>) {
    hipError_t r = hipErrorInvalidValue;
    bool hit = ((a.D == 32 + 8 * Ds ? (r = launch_short_d<ET, 32 + 8 * Ds>(a), true) : false) || ...);
    return hit ? r : hipErrorInvalidValue;
}

}  // namespace

bool attn_fwd_short_supported(int D, int Lk) {
    // D from 32 to 160 in steps of 8; up to four 32-key sub-tiles
    return Lk >= 1 && Lk <= 128 && D >= 32 && D <= 160 && D % 8 == 0;
}

hipError_t launch_attn_fwd_short(const AttnArgs& a) {
    using Seq = std::make_integer_sequence<int, 17>;   // D = 32, 40, ..., 160
    return a.dtype == kF16 ? dispatch_short<kF16>(a, Seq{}) : dispatch_short<kBF16>(a, Seq{});
}

}  // namespace sdattn
