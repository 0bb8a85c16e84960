// attn_fwd_generic.hip -- single-pass attention forward (Eq. 3) for gfx950,
// generic over the head width (any D % 8 == 0 up to 256).  Used for the head
// widths the LDS-streaming kernel does not cover (D < 32, or D too wide for
// its buffers); the algorithm is the same.
//
// One workgroup = 4 waves = 128 query rows of one (batch, head); each wave
// owns 32 rows.  Keys and values stream through LDS in tiles of 64 keys,
// double buffered (global loads of tile t+1 are in flight while tile t is
// consumed).  Per tile and wave:
//
//   S^T = K Q^T      32x32x16 MFMA, A = K tile from LDS, B = Q^T held in
//                    registers for the whole kernel; the accumulator puts one
//                    query per lane (lane % 32) and 16 of the 32 keys of a
//                    sub-tile in that lane's registers, so the row max needs
//                    one exchange between the lane halves (v_permlane32_swap).
//   p = 2^(c s - m)  c = |scale| log2(e); m is a running reference that is
//                    only moved (with the matching rescale of O and l) when a
//                    tile's maximum exceeds it by more than 15, and then to
//                    that maximum less 8: p <= 2^15 always, the largest
//                    weights near 2^8, and weights down to 2^-32 of them
//                    above fp16's smallest subnormal.
//   O^T += V^T P^T   32x32x16 MFMA, A = V^T from a transposed LDS tile, B = P
//                    straight from the S^T accumulator registers (no shuffle);
//                    O^T again has one query per lane.
//   l                the row sum of the rounded p.  When D is not a multiple of
//                    32 the padding rows of V^T carry a row of ones at d = D, so
//                    the P V product yields l in O^T[D]; otherwise the packed p
//                    pairs are summed with v_dot2 against (1, 1).
//
// This is the "multi-stage" reduction of Sec. 3.2.1 (a per-tile max and
// exponential sum merged into the running pair) fused with the element-wise
// normalisation and the product with V, so the N x M matrix A is never
// written (FlashAttention's tiling, Sec. 3.2.2).
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kBQ = kWaves * 32;   // query rows per workgroup
constexpr int kKB = 64;            // keys per LDS tile
constexpr int kVS = kKB + 4;       // V^T row pitch in elements (conflict-free 8-byte reads)
constexpr float kPBias = 8.0f;          // m = a logit maximum less this
constexpr float kRescaleLimit = 15.0f;  // largest weight before m moves: 2^15

// K tile row pitch (elements): D rounded so that pitch/8 is odd, which keeps
// the 16-byte reads of 16 consecutive rows on distinct LDS banks.
__host__ __device__ constexpr int k_pitch(int D) { return ((D / 8) & 1) ? D : D + 8; }

template <int ET, int DK>
__global__ __launch_bounds__(kThreads) void attn_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    uint16_t* __restrict__ O, float* __restrict__ LS, int Lq, int Lk, int D, float scale_abs,
    float c, int neg, int nqb, int oh) {
    constexpr int DN = (DK + 1) / 2;       // 32-wide d tiles of O^T
    constexpr int DNP = DN * 32;           // padded d rows of V^T
    constexpr int KCH = (kKB * 2 * DK + kThreads - 1) / kThreads;        // 16-byte K chunks per thread
    constexpr int VCH = ((kKB / 2) * 2 * DK + kThreads - 1) / kThreads;  // V key-pair tasks per thread

    extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
    const int KP = k_pitch(D);
    uint16_t* Ks = smem;                         // [2][kKB][KP]
    uint16_t* Vt = smem + 2 * kKB * KP;          // [2][DNP][kVS]

    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = tid >> 6;

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int bh = tile / nqb;
    const int qb = tile - bh * nqb;
    const int q0 = qb * kBQ + wave * 32;

    const uint16_t* Qh = Q + (size_t)bh * Lq * D;
    const uint16_t* Kh = K + (size_t)bh * Lk * D;
    const uint16_t* Vh = V + (size_t)bh * Lk * D;
    const bool ones_row = (D % 32) != 0;

    // Constant padding rows of V^T (d >= D): a row of ones at d = D when it
    // exists (it turns the P V product into the row sum), zeros elsewhere.
    // Tile stores only ever write rows d < D, so this is done once.
    for (int i = tid; i < 2 * (DNP - D) * kVS; i += kThreads) {
        const int b = i / ((DNP - D) * kVS);
        const int rr = i - b * (DNP - D) * kVS;
        const int d = D + rr / kVS;
        Vt[(size_t)b * DNP * kVS + d * kVS + rr % kVS] =
            (d == D) ? from_float<ET>(1.0f) : (uint16_t)0;
    }

    // Q^T operand: lane holds query q0 + l32, d = 16s + 8*half .. +7 for each s.
    const int qrow = q0 + l32;
    u32x4 qreg[DK];
#pragma unroll
    for (int s = 0; s < DK; ++s) {
        const int d0 = 16 * s + 8 * half;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (qrow < Lq && d0 < D) v = *(const u32x4*)(Qh + (size_t)qrow * D + d0);
        if (neg) v ^= 0x80008000u;   // fold a negative scale into Q (exact)
        qreg[s] = v;
    }

    // Per-thread share of a tile load; the mapping is the same for every tile.
    const int DC = D / 8;                  // 16-byte chunks per row
    int k_goff[KCH], k_loff[KCH], k_key[KCH];
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
        const int ci = tid + i * kThreads;
        const int key = ci / DC, cc = ci - key * DC;
        k_key[i] = ci < kKB * DC ? key : kKB;   // kKB marks "no chunk"
        k_goff[i] = key * D + 8 * cc;
        k_loff[i] = key * KP + 8 * cc;
    }
    int v_key[VCH], v_goff[VCH], v_loff[VCH];
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
        const int ti = tid + i * kThreads;
        const int kp = ti % (kKB / 2), cc = ti / (kKB / 2);
        v_key[i] = ti < (kKB / 2) * DC ? 2 * kp : kKB;
        v_goff[i] = 2 * kp * D + 8 * cc;
        v_loff[i] = 8 * cc * kVS + 2 * kp;
    }

    u32x4 kbuf[KCH], vbuf0[VCH], vbuf1[VCH];
    auto load_tile = [&](int kbase) {
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (k_key[i] < kKB && kbase + k_key[i] < Lk)
                v = *(const u32x4*)(Kh + (size_t)kbase * D + k_goff[i]);
            kbuf[i] = v;
        }
#pragma unroll
        for (int i = 0; i < VCH; ++i) {
            u32x4 a = {0u, 0u, 0u, 0u}, b = {0u, 0u, 0u, 0u};
            if (v_key[i] < kKB) {
                if (kbase + v_key[i] < Lk) a = *(const u32x4*)(Vh + (size_t)kbase * D + v_goff[i]);
                if (kbase + v_key[i] + 1 < Lk) b = *(const u32x4*)(Vh + (size_t)kbase * D + v_goff[i] + D);
            }
            vbuf0[i] = a;
            vbuf1[i] = b;
        }
    };
    auto store_tile = [&](int buf) {
        uint16_t* kd = Ks + buf * kKB * KP;
        uint16_t* vd = Vt + buf * DNP * kVS;
#pragma unroll
        for (int i = 0; i < KCH; ++i)
            if (k_key[i] < kKB) *(u32x4*)(kd + k_loff[i]) = kbuf[i];
#pragma unroll
        for (int i = 0; i < VCH; ++i) {
            if (v_key[i] < kKB) {
                // transpose: element e of the two keys' chunks goes to row 8*cc + e
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const uint32_t x = vbuf0[i][w], y = vbuf1[i][w];
                    *(uint32_t*)(vd + v_loff[i] + (2 * w) * kVS) = (x & 0xffffu) | (y << 16);
                    *(uint32_t*)(vd + v_loff[i] + (2 * w + 1) * kVS) = (x >> 16) | (y & 0xffff0000u);
                }
            }
        }
    };

    f32x16 acc[DN];
#pragma unroll
    for (int n = 0; n < DN; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[n][r] = 0.0f;
    float m_run = -__builtin_inff();   // running max used in the exponent (log2 units)
    float s_max = -__builtin_inff();   // true running max of the raw scores
    float l_part = 0.0f;               // this lane's part of the row sum (vector-ALU path)

    const int nkb = (Lk + kKB - 1) / kKB;
    load_tile(0);
    store_tile(0);
    __syncthreads();

    for (int kb = 0; kb < nkb; ++kb) {
        const int kbase = kb * kKB;
        const int buf = kb & 1;
        if (kb + 1 < nkb) load_tile(kbase + kKB);

        const uint16_t* kt = Ks + buf * kKB * KP;
        const uint16_t* vt = Vt + buf * DNP * kVS;

        // ---- S^T = K Q^T for the tile's two 32-key sub-tiles
        f32x16 st[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int r = 0; r < 16; ++r) st[t][r] = 0.0f;
#pragma unroll
            for (int s = 0; s < DK; ++s) {
                const int d0 = 16 * s + 8 * half;
                u32x4 a = {0u, 0u, 0u, 0u};
                if (d0 < D) a = *(const u32x4*)(kt + (32 * t + l32) * KP + d0);
                st[t] = mfma32x32x16<ET>(a, qreg[s], st[t]);
            }
        }

        // ---- masking of keys past Lk (last tile only)
        const bool tail = kbase + kKB > Lk;
        if (tail) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kbase + 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (key >= Lk) st[t][r] = -__builtin_inff();
                }
        }

        // ---- row maximum of the tile (Eq. 4's L, one stage of the merge)
        float mloc = st[0][0];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, st[t][r]);
        mloc = half_max(mloc);
        s_max = fmaxf(s_max, mloc);
        const float mb = mloc * c;
        if (__any(mb > m_run + kRescaleLimit)) {
            const float m_new = fmaxf(m_run, mb - kPBias);
            const float alpha = fast_exp2(m_run - m_new);
#pragma unroll
            for (int n = 0; n < DN; ++n)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[n][r] *= alpha;
            l_part *= alpha;
            m_run = m_new;
        }

        // ---- p = 2^(c s - m), rounded to the input type, as the B operand
        const float negm = -m_run;
        u32x4 pk[2][2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            float p[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) p[r] = fast_exp2(fmaf(st[t][r], c, negm));
            if (tail) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kbase + 32 * t + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (key >= Lk) p[r] = 0.0f;
                }
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w) pk[t][u][w] = pack2<ET>(p[8 * u + 2 * w], p[8 * u + 2 * w + 1]);
            if (!ones_row) {
                // sum the rounded p, so numerator and denominator use the same weights
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int w = 0; w < 4; ++w) l_part = add_pair<ET>(pk[t][u][w], l_part);
            }
        }

        // ---- O^T += V^T P^T
#pragma unroll
        for (int n = 0; n < DN; ++n) {
            const uint16_t* vrow = vt + (32 * n + l32) * kVS;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int col = 32 * t + 16 * u + 4 * half;
                    const u32x2 lo = *(const u32x2*)(vrow + col);
                    const u32x2 hi = *(const u32x2*)(vrow + col + 8);
                    const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                    acc[n] = mfma32x32x16<ET>(a, pk[t][u], acc[n]);
                }
        }

        if (kb + 1 < nkb) store_tile(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: l, O / l, store
    float l;
    if (ones_row) {
        const int dd = D % 32;                         // position of the ones row in its d tile
        const int hsel = (dd >> 2) & 1, rsel = 4 * (dd >> 3) + (dd & 3);
        const int nsel = D / 32;
        float own = 0.0f;
#pragma unroll
        for (int n = 0; n < DN; ++n)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (n == nsel && r == rsel) own = acc[n][r];
        const float other = half_partner(own, half);
        l = (half == hsel) ? own : other;
    } else {
        l = half_sum(l_part);
    }
    const float inv = 1.0f / l;
    if (qrow < Lq) {
        uint16_t* orow = out_base(O, bh, Lq, D, oh) + (size_t)qrow * out_stride(D, oh);
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
            const float Lrow = s_max * scale_abs;
            const float Srow = l * fast_exp2(m_run - s_max * c);
            float* o2 = LS + ((size_t)bh * Lq + qrow) * 2;
            o2[0] = Lrow;
            o2[1] = Srow;
        }
    }
}

// LDS of the widest D that maps to DK (D = 16*DK)
template <int DK>
constexpr size_t max_lds_bytes() {
    return (size_t)2 * kKB * k_pitch(16 * DK) * 2 + (size_t)2 * (((DK + 1) / 2) * 32) * kVS * 2;
}

template <int ET, int DK>
hipError_t launch_dk(const AttnArgs& a) {
    const int nqb = (a.Lq + kBQ - 1) / kBQ;
    const long long nblk = (long long)a.B * a.H * nqb;
    const int KP = k_pitch(a.D);
    constexpr int DNP = ((DK + 1) / 2) * 32;
    const size_t lds = (size_t)2 * kKB * KP * 2 + (size_t)2 * DNP * kVS * 2;
    const float scale_abs = a.scale < 0 ? -a.scale : a.scale;
    const float c = scale_abs * kLog2e;
    // allow the dynamic LDS of the widest heads (above 64 KiB); done once per instantiation
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&attn_fwd_kernel<ET, DK>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)max_lds_bytes<DK>());
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL((attn_fwd_kernel<ET, DK>), dim3((unsigned)nblk), dim3(kThreads), lds,
                       (hipStream_t)a.stream, (const uint16_t*)a.q, (const uint16_t*)a.k,
                       (const uint16_t*)a.v, (uint16_t*)a.out, a.ls, a.Lq, a.Lk, a.D, scale_abs, c,
                       a.scale < 0 ? 1 : 0, nqb, a.o_rows ? a.H : 0);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_et(const AttnArgs& a) {
    switch ((a.D + 15) / 16) {
        case 1: return launch_dk<ET, 1>(a);
        case 2: return launch_dk<ET, 2>(a);
        case 3: return launch_dk<ET, 3>(a);
        case 4: return launch_dk<ET, 4>(a);
        case 5: return launch_dk<ET, 5>(a);
        case 6: return launch_dk<ET, 6>(a);
        case 7: return launch_dk<ET, 7>(a);
        case 8: return launch_dk<ET, 8>(a);
        case 9: return launch_dk<ET, 9>(a);
        case 10: return launch_dk<ET, 10>(a);
        case 11: return launch_dk<ET, 11>(a);
        case 12: return launch_dk<ET, 12>(a);
        case 13: return launch_dk<ET, 13>(a);
        case 14: return launch_dk<ET, 14>(a);
        case 15: return launch_dk<ET, 15>(a);
        case 16: return launch_dk<ET, 16>(a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_attn_fwd_generic(const AttnArgs& a) {
    return a.dtype == kF16 ? launch_et<kF16>(a) : launch_et<kBF16>(a);
}

}  // namespace sdattn
