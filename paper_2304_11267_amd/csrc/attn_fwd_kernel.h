// attn_fwd_kernel.h -- single-pass attention forward (Eq. 3) for gfx950, with the
// K and V tiles streamed into LDS by direct global->LDS copies.
//
// One workgroup covers 128 query rows of one (batch, head) (64 or 256 in the
// other geometries, see Geom).  Its waves are
// split in two halves over the key tiles (the first half of the tiles and the
// second; four quarters in one geometry), and at the end the parts of every
// row are merged through LDS.
// A wave owns QB blocks of 32 query rows: QB = 2 when D <= 64 (4 waves per
// 128-row workgroup), QB = 1 above (8 waves).  With QB = 2 every K and V^T operand
// read from LDS feeds two MFMAs.  Registers are budgeted for two waves per
// SIMD (256 each), or for one (up to 512) where the LDS already limits a CU
// to one wave per SIMD.
// Key/value tiles of 64 keys (128 with 256-row workgroups) move through LDS
// double-buffered per half: while
// one tile is consumed the next is copied straight from global memory
// (global_load_lds, 16 bytes per lane, no registers involved), keeping the
// row-major [key][d] layout.  Per 32-key sub-tile, wave and query block:
//
//   S^T = K Q^T      32x32x16 MFMA.  A = K rows read from LDS (16 bytes per
//                    lane), B = Q^T held in registers for the whole kernel.
//                    The accumulator puts one query per lane (lane % 32) and
//                    16 of the 32 keys in that lane, so the row maximum needs a
//                    single exchange between lane halves.
//   p = 2^(c s - m)  c = |scale| log2(e), one FMA and one exponential per
//                    score.  m is fixed at the maximum of each wave's first
//                    sub-tile less kPBias = 8 (p may then exceed 1); a row
//                    whose later logits would overflow the rounded p sends the
//                    workgroup through an exact fallback in which m moves, with
//                    the rescale of O and l, whenever a weight would pass 2^15.
//                    The bias keeps the largest weights near 2^8 instead of 1,
//                    so weights down to 2^-32 of the largest survive rounding
//                    to fp16 (its subnormals end at 2^-24): on very long key
//                    sequences their sum is otherwise lost.
//   O^T += V^T P^T   32x32x16 MFMA.  B = P straight from the S^T registers;
//                    A = V^T, produced from the row-major V tile by the
//                    transposing LDS read ds_read_b64_tr_b16: 16 lanes each
//                    point at 4 consecutive d of one key, and every lane gets
//                    4 consecutive keys of one d.
//   l                row sum of the rounded p.  When D is not a multiple of 32
//                    (and the LDS has room for it), the lanes whose d lies past
//                    D read a constant block instead of V: a one at d = D and
//                    zeros beyond, so the P V product also yields l in row D of
//                    O^T.  Otherwise the packed p pairs are summed with v_dot2
//                    against (1, 1).
//
// With the maximum fixed, a whole 64-key tile is written as a software
// pipeline, so that each step's softmax has the independent MFMAs of its
// neighbours beside it, and left to the compiler's scheduler.
//
// This is the block-wise ("multi-stage") reduction of Sec. 3.2.1 -- a block's
// maximum and exponential sum merged into the running pair, and the key
// halves merged by the same rule -- fused with the element-wise normalisation
// and the product with V, so the N x M matrix A never leaves the chip (the
// IO-aware tiling of FlashAttention, Sec. 3.2.2).
//
// The kernel templates live in this header; attn_fwd.hip instantiates them
// for fp16 (and holds the entry points), attn_fwd_bf16.hip for bf16, so the
// two halves compile in parallel.
#pragma once

#include <utility>

#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

// Workgroup geometries (the GEO template argument): rows of queries per
// workgroup and keys per LDS tile.
constexpr int kGeoSmall = 0;           // 64 rows, 64-key tiles
constexpr int kGeoNormal = 1;          // 128 rows, 64-key tiles
constexpr int kGeoBig = 2;             // 256 rows, 128-key tiles (QB = 2 only)
constexpr int kGeoQuarter = 3;         // 64 rows, keys split four ways, 64-key tiles
// The exponent's reference m sits kPBias below the logit maximum it was
// taken from (weights of the largest logits near 2^8; see p = 2^(c s - m)
// above); the online path moves m once a sub-tile's maximum would give a
// weight above 2^kRescaleLimit (fp16 holds values below 2^16).
constexpr float kPBias = 8.0f;
constexpr float kRescaleLimit = 15.0f;
constexpr int kMaxLds = 160 * 1024;
constexpr int kQuarterMinKeys = 512;   // shortest key sequence given to kGeoQuarter

// QB = 32-row query blocks per wave.  With QB = 2 every K and V^T operand
// read from LDS feeds two MFMAs (half the LDS traffic per flop) and each wave
// carries two independent MFMA / softmax chains; the register budget is then
// sized for two waves per SIMD.
//
// kGeoSmall halves the query waves of a workgroup (64 query rows instead of
// 128), for calls whose 128-row blocks would leave CUs idle (fewer than 256
// workgroups: the 32x32 and 16x16 levels).  kGeoBig doubles them (256 rows,
// eight waves) and the keys per tile (128), for grids that still cover the
// CUs: each K/V tile then serves twice the queries and a barrier twice the
// keys, in the LDS the two 128-row workgroups of a CU would otherwise hold.
// kGeoQuarter keeps kGeoSmall's 64 rows but splits the keys four ways
// instead of two (eight waves), for small grids whose LDS would otherwise
// leave one wave per SIMD: two waves then share each SIMD and hide each
// other's MFMA and exponential latencies.  Its tiles carry no constant
// block (the LDS holds four splits' double buffers), so l comes from v_dot2.
template <int D, int GEO = kGeoNormal>
struct Geom {
    static constexpr int QB = D <= 64 ? 2 : 1;
    static constexpr bool kBig = GEO == kGeoBig;
    static constexpr bool kQuarter = GEO == kGeoQuarter;
    static constexpr int kKS = kQuarter ? 4 : 2;              // key splits
    static constexpr int kTK = kBig ? 128 : 64;               // keys per LDS tile
    static constexpr int kQW = kBig ? 4 : (GEO == kGeoSmall || kQuarter ? 2 : 4) / QB;   // query waves
    static constexpr int kBQ = 32 * QB * kQW;                 // query rows per workgroup
    static constexpr int kWaves = kKS * kQW;                  // times the key splits
    static constexpr int kThreads = kWaves * 64;
    static constexpr int DK = (D + 15) / 16;                  // 16-deep k steps of Q K^T
    static constexpr int DN = (D + 31) / 32;                  // 32-row d tiles of O^T
    static constexpr bool kOnes = (D % 32) != 0 && !kQuarter;   // padding rows carry the row sum
    static constexpr int kTileBytes = kTK * D * 2;            // one K or V tile
    static constexpr int kChunks = kTileBytes / 1024;         // 1 KiB wave copies per tile
    static constexpr int kBufBytes = kTileBytes * (kOnes ? 3 : 2);   // K, V (, constant block)
    static constexpr int kHalfBytes = 2 * kBufBytes;          // two buffers per key split
    static constexpr int kMergeFloats = QB * (DN * 16 * 64 + 3 * 64);   // one wave's O^T, m, max, l
    static constexpr int kMergeBytes = (kKS - 1) * kQW * kMergeFloats * 4;
    static constexpr int kLdsBytes = kKS * kHalfBytes > kMergeBytes ? kKS * kHalfBytes : kMergeBytes;
    static constexpr bool kFits = D >= 32 && D % 8 == 0 && kLdsBytes <= kMaxLds && (!kBig || QB == 2);
    // Waves per SIMD the register budget is sized for: two (256 registers
    // each) when the LDS lets enough workgroups share a CU, else one, which
    // leaves a wave up to 512 registers (the matrix-core registers then take
    // what would otherwise spill to scratch) at no cost in occupancy.
    static constexpr int kWgPerCu = kLdsBytes <= kMaxLds ? kMaxLds / kLdsBytes : 1;
    static constexpr int kWavesPerSimd = kWgPerCu * kWaves >= 8 ? 2 : 1;
};

template <int ET, int D, bool STATS, bool OROWS, int GEO>
__global__ __launch_bounds__((Geom<D, GEO>::kThreads), (Geom<D, GEO>::kWavesPerSimd)) void attn_fwd_lds_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
    uint16_t* __restrict__ O, float* __restrict__ LS, int Lq, int Lk, float scale_abs, float c,
    int neg, int nqb, int oh) {
    using G = Geom<D, GEO>;
    constexpr int DK = G::DK;
    constexpr int DN = G::DN;
    constexpr int QB = G::QB;
    constexpr int kQW = G::kQW;
    constexpr int kWaves = G::kWaves;
    constexpr int kThreads = G::kThreads;
    constexpr int TB = G::kTileBytes;

    extern __shared__ __attribute__((aligned(16))) char smem[];

    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kh = wave / kQW;         // key split ("half" when there are two) of this wave
    const int wq = wave % kQW;         // query slot of this wave

    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int bh = tile / nqb;
    const int qb = tile - bh * nqb;
    const int q0 = qb * G::kBQ + wq * 32 * QB;   // first row of this wave's QB blocks

    const char* Kh = (const char*)(K + (size_t)bh * Lk * D);
    const char* Vh = (const char*)(V + (size_t)bh * Lk * D);
    char* hbase = smem + kh * G::kHalfBytes;   // this split's two buffers

    // Constant blocks (one per buffer): a one in column 0 of every row, zeros
    // elsewhere.  Lanes whose d lies at or past D read these instead of V.
    if constexpr (G::kOnes) {
        const uint32_t one = from_float<ET>(1.0f);
        for (int i = tid; i < 2 * G::kKS * (TB / 16); i += kThreads) {
            const int b = i / (TB / 16), j = i - b * (TB / 16);
            u32x4 w = {0u, 0u, 0u, 0u};
            if ((j * 8) % D == 0) w[0] = one;
            *(u32x4*)(smem + b * G::kBufBytes + 2 * TB + j * 16) = w;
        }
    }

    // Tiles of this split: [t_first, t_first + t_count).  Split s takes
    // tiles s * nh .. s * nh + nh - 1 (nh = ceil(ntiles / kKS)), the last
    // ones what remains, possibly none; all run nh steps.
    constexpr int kTK = G::kTK;
    const int ntiles = (Lk + kTK - 1) / kTK;
    const int nh = (ntiles + G::kKS - 1) / G::kKS;
    const int t_first = kh * nh;
    const int t_count = min(nh, max(0, ntiles - t_first));

    // Copy tile t of this split into its buffer b (the split's kQW waves issue
    // the 1 KiB pieces wq, wq + kQW, ...).  Rows past Lk repeat row Lk - 1
    // (finite data; their weights are forced to zero).
    auto issue_tile = [&](int t, int b) __attribute__((always_inline)) {
        const int kbase = t * kTK;
        char* bufp = hbase + b * G::kBufBytes;
        if (kbase + kTK <= Lk) {
            // a full tile is one contiguous run of K (and of V) rows; byte
            // offsets inside a head fit 32 bits (the launch checks Lk * D)
            const uint32_t tile_off = (uint32_t)kbase * (2 * D) + lane * 16;
#pragma unroll
            for (int i = 0; i < (2 * G::kChunks + kQW - 1) / kQW; ++i) {
                const int cidx = wq + kQW * i;
                if (cidx < 2 * G::kChunks) {
                    const bool isv = cidx >= G::kChunks;
                    const int cc = isv ? cidx - G::kChunks : cidx;
                    const char* src = isv ? Vh : Kh;
                    __builtin_amdgcn_global_load_lds(src + (size_t)(tile_off + cc * 1024),
                                                     (lds_void_t*)(bufp + (isv ? TB : 0) + cc * 1024),
                                                     16, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < (2 * G::kChunks + kQW - 1) / kQW; ++i) {
                const int cidx = wq + kQW * i;
                if (cidx < 2 * G::kChunks) {
                    const bool isv = cidx >= G::kChunks;
                    const int cc = isv ? cidx - G::kChunks : cidx;
                    const int byte = cc * 1024 + lane * 16;
                    const int row = byte / (2 * D);
                    const int col = byte - row * (2 * D);
                    const size_t goff = (size_t)min(kbase + row, Lk - 1) * (2 * D) + col;
                    __builtin_amdgcn_global_load_lds((isv ? Vh : Kh) + goff,
                                                     (lds_void_t*)(bufp + (isv ? TB : 0) + cc * 1024),
                                                     16, 0, 0);
                }
            }
        }
    };

    // Q^T operand of block j: lane holds query q0 + 32j + l32, d = 16s + 8*half .. +7.
    u32x4 qreg[QB][DK];
#pragma unroll
    for (int j = 0; j < QB; ++j)
#pragma unroll
        for (int s = 0; s < DK; ++s) {
            const int qrow = q0 + 32 * j + l32;
            const int d0 = 16 * s + 8 * half;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (qrow < Lq && d0 < D) v = *(const u32x4*)(Q + ((size_t)bh * Lq + qrow) * D + d0);
            if (neg) v ^= 0x80008000u;   // fold a negative scale into Q (exact)
            qreg[j][s] = v;
        }


    // Per-lane LDS byte offsets inside a buffer.
    // K rows: lane reads key row l32 at d = 8*half (+16 s, +32 sub rows).
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
            // past D: the constant block, or (without one) V columns 32
            // lower, whose finite products land in O^T rows never stored
            v_off[n] = ds < D ? TB + (krow * D + ds) * 2
                              : G::kOnes ? 2 * TB + (krow * D + ds - D) * 2 : TB + (krow * D + ds - 32) * 2;
        }
    }

    f32x16 acc[QB][DN];
    float m_run[QB];   // running max used in the exponent (log2 units)
    float s_max[QB];   // true running max of the raw scores
    float l_part[QB];  // this lane's part of the row sum (v_dot2 path)
    auto reset = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < QB; ++j) {
#pragma unroll
            for (int n = 0; n < DN; ++n)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[j][n][r] = 0.0f;
            m_run[j] = -__builtin_inff();
            s_max[j] = -__builtin_inff();
            l_part[j] = 0.0f;
        }
    };
    reset();

    // How a sub-tile treats the running maximum m (log2 units):
    //   kFirst  the wave's first sub-tile: m = its row maximum - kPBias (O is
    //           still 0)
    //   kFixed  m stays; p = 2^(c s - m) may exceed 1, and if a later logit
    //           exceeds the first sub-tile's maximum by more than ~8 the
    //           rounded p overflows to inf, which the overflow vote after the
    //           loop detects
    //   kOnline m moves (with the rescale of O and l) to a sub-tile's maximum
    //           - kPBias whenever that maximum exceeds m by more than
    //           kRescaleLimit -- the fallback
    enum { kFirst = 0, kFixed = 1, kOnline = 2 };

    // One 32-key sub-tile (keys kbase ..) held at row offset `sub` * 32 of
    // the tile in buffer base `buf`.
    auto step32 = [&](auto mode_c, auto tail_c, const char* buf, int sub, int kbase)
                      __attribute__((always_inline)) {
        constexpr int MODE = decltype(mode_c)::value;
        constexpr bool TAIL = decltype(tail_c)::value;
        // ---- S^T = K Q^T, one K operand read for the QB blocks
        f32x16 st[QB];
#pragma unroll
        for (int j = 0; j < QB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) st[j][r] = 0.0f;
#pragma unroll
        for (int s = 0; s < DK; ++s) {
            u32x4 a = *(const u32x4*)(buf + k_off + (32 * sub * D + 16 * s) * 2);
#pragma unroll
            for (int j = 0; j < QB; ++j) st[j] = mfma32x32x16<ET>(a, qreg[j][s], st[j]);
        }
        u32x4 pk[QB][2];
#pragma unroll
        for (int j = 0; j < QB; ++j) {
            if constexpr (TAIL) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kbase + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (key >= Lk) st[j][r] = -__builtin_inff();
                }
            }
            // ---- row maximum (Eq. 4's L), where the mode needs it
            if constexpr (MODE != kFixed || STATS) {
                float mloc = st[j][0];
#pragma unroll
                for (int r = 1; r < 16; ++r) mloc = fmaxf(mloc, st[j][r]);
                mloc = half_max(mloc);
                s_max[j] = fmaxf(s_max[j], mloc);
                if constexpr (MODE == kFirst) {
                    m_run[j] = mloc * c - kPBias;
                } else if constexpr (MODE == kOnline) {
                    const float mb = mloc * c;
                    if (__any(mb > m_run[j] + kRescaleLimit)) {
                        const float m_new = fmaxf(m_run[j], mb - kPBias);
                        const float alpha = fast_exp2(m_run[j] - m_new);
#pragma unroll
                        for (int n = 0; n < DN; ++n)
#pragma unroll
                            for (int r = 0; r < 16; ++r) acc[j][n][r] *= alpha;
                        l_part[j] *= alpha;
                        m_run[j] = m_new;
                    }
                }
            }
            // ---- p = 2^(c s - m), rounded to the input type
            const float negm = -m_run[j];
            float p[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) p[r] = fast_exp2(fmaf(st[j][r], c, negm));
            if constexpr (TAIL) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kbase + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (key >= Lk) p[r] = 0.0f;
                }
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    pk[j][u][w] = pack2<ET>(p[8 * u + 2 * w], p[8 * u + 2 * w + 1]);
            if constexpr (!G::kOnes) {
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int w = 0; w < 4; ++w) l_part[j] = add_pair<ET>(pk[j][u][w], l_part[j]);
            }
        }
        // ---- O^T += V^T P^T; keys of operand slot e: 16u + 8*(e/4) + 4*half + e%4
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int n = 0; n < DN; ++n) {
                const char* vb = buf + v_off[n] + (32 * sub + 16 * u) * D * 2;
                const u32x2 lo = lds_read_tr(vb);
                const u32x2 hi = lds_read_tr(vb + 8 * D * 2);
                const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
#pragma unroll
                for (int j = 0; j < QB; ++j) acc[j][n] = mfma32x32x16<ET>(a, pk[j][u], acc[j][n]);
            }
    };

    std::integral_constant<bool, false> full_c;
    std::integral_constant<bool, true> tail_c;
    std::integral_constant<int, kFirst> first_c;
    std::integral_constant<int, kFixed> fixed_c;
    std::integral_constant<int, kOnline> online_c;

    // A whole 64-key tile with the maximum fixed, written as a software
    // pipeline over the (sub-tile, block) pairs P0 = (0, 0), P1 = (0, 1), ...:
    //   S^T of sub-tile 0, then S^T of sub-tile 1 beside the softmax of P0,
    //   then the P V product of P(k-1) beside the softmax of Pk, and last
    //   the P V product of the last pair
    // so that each softmax has independent MFMAs next to it.  The compiler
    // schedules the whole tile: fences between these steps, or exponentials
    // pinned between the MFMAs, measured 1-2 % slower.
    auto tile_fixed = [&](const char* buf) __attribute__((always_inline)) {
        constexpr int NP = 2 * QB;               // (sub-tile, block) pairs
        f32x16 st[2][QB];
        u32x4 pk[2][QB][2];
        u32x4 vt[2][2][DN];
        auto qk = [&](int sub) __attribute__((always_inline)) {
#pragma unroll
            for (int j = 0; j < QB; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) st[sub][j][r] = 0.0f;
#pragma unroll
            for (int s = 0; s < DK; ++s) {
                u32x4 a = *(const u32x4*)(buf + k_off + (32 * sub * D + 16 * s) * 2);
    #pragma unroll
                for (int j = 0; j < QB; ++j) st[sub][j] = mfma32x32x16<ET>(a, qreg[j][s], st[sub][j]);
            }
        };
        auto read_vt = [&](int sub) __attribute__((always_inline)) {
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int n = 0; n < DN; ++n) {
                    const char* vb = buf + v_off[n] + (32 * sub + 16 * u) * D * 2;
                    const u32x2 lo = lds_read_tr(vb);
                    const u32x2 hi = lds_read_tr(vb + 8 * D * 2);
                    vt[sub][u][n] = u32x4{lo[0], lo[1], hi[0], hi[1]};
                }
        };
        auto softmax = [&](int pr) __attribute__((always_inline)) {
            const int sub = pr / QB, j = pr % QB;
            float p[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) p[r] = fast_exp2(fmaf(st[sub][j][r], c, -m_run[j]));
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    pk[sub][j][u][w] = pack2<ET>(p[8 * u + 2 * w], p[8 * u + 2 * w + 1]);
            if constexpr (!G::kOnes) {
#pragma unroll
                for (int u = 0; u < 2; ++u)
#pragma unroll
                    for (int w = 0; w < 4; ++w) l_part[j] = add_pair<ET>(pk[sub][j][u][w], l_part[j]);
            }
        };
        auto pv = [&](int pr) __attribute__((always_inline)) {
            const int sub = pr / QB, j = pr % QB;
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int n = 0; n < DN; ++n) acc[j][n] = mfma32x32x16<ET>(vt[sub][u][n], pk[sub][j][u], acc[j][n]);
        };
        qk(0);
        qk(1);
        read_vt(0);
        softmax(0);
#pragma unroll
        for (int k = 1; k < NP; ++k) {
            if (k == QB) read_vt(1);
            pv(k - 1);
            softmax(k);
        }
        if (QB == 1) read_vt(1);
        pv(NP - 1);
    };

    // consume the tile t (in buffer b) of this half; its first sub-tile in
    // mode mode0_c, the others in mode_c.  A pipelined 64-key step reads its
    // rows relative to the pointer it gets, so a 128-key tile is two of them.
    auto consume = [&](auto mode0_c, auto mode_c, int t, int b) __attribute__((always_inline)) {
        const char* buf = hbase + b * G::kBufBytes;
        const int kbase = t * kTK;
        constexpr bool kPipelined = decltype(mode0_c)::value == kFixed &&
                                    decltype(mode_c)::value == kFixed && !STATS;
        if (kbase + kTK <= Lk) {
            if constexpr (kPipelined) {
#pragma unroll
                for (int h = 0; h < kTK / 64; ++h) tile_fixed(buf + h * 64 * D * 2);
            } else {
                step32(mode0_c, full_c, buf, 0, kbase);
#pragma unroll
                for (int sb = 1; sb < kTK / 32; ++sb) step32(mode_c, full_c, buf, sb, kbase + 32 * sb);
            }
        } else {
            if (kbase + 32 <= Lk) step32(mode0_c, full_c, buf, 0, kbase);
            else step32(mode0_c, tail_c, buf, 0, kbase);
#pragma unroll
            for (int sb = 1; sb < kTK / 32; ++sb) {
                const int kb = kbase + 32 * sb;
                if (kb + 32 <= Lk) step32(mode_c, full_c, buf, sb, kb);
                else if (kb < Lk) step32(mode_c, tail_c, buf, sb, kb);
            }
        }
    };

    // The 64-key half h of the whole tile t (buffer b) of a 128-key geometry
    // on the pipelined path.
    auto consume_half = [&](int b, int h) __attribute__((always_inline)) {
        tile_fixed(hbase + b * G::kBufBytes + h * 64 * D * 2);
    };

    // all tiles of this half: the first tile opens with kFirst, every other
    // sub-tile runs in mode_c (kFixed, or kOnline for the fallback)
    auto run_tiles = [&](auto mode_c) __attribute__((always_inline)) {
        if (t_count > 0) issue_tile(t_first, 0);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (t_count > 0) {
            if (t_count > 1) issue_tile(t_first + 1, 1);
            consume(first_c, mode_c, t_first, 0);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        // Inside the loop only whole tiles are consumed; a ragged last tile
        // (the last tile of its half: nothing is copied over it afterwards)
        // waits in its buffer until the loop ends.  With a single way through
        // the loop body the accumulators keep their registers across
        // iterations instead of being copied at a join.
        // With 128-key tiles on the fixed-maximum path the workgroup also
        // meets between the two 64-key halves of every tile (faster at the
        // 64x64 level while the tile's steps were fenced, neutral since);
        // that barrier sits outside the conditions so every wave of both key
        // halves reaches it.
        constexpr bool kMidBarrier = G::kBig && decltype(mode_c)::value == kFixed && !STATS;
        int pend = -1;
        for (int i = 1; i < nh; ++i) {
            const int b = i & 1;
            if (i + 1 < t_count) issue_tile(t_first + i + 1, b ^ 1);
            if constexpr (kMidBarrier) {
                const bool whole = i < t_count && (t_first + i + 1) * kTK <= Lk;
                if (i < t_count && !whole) pend = i;
                if (whole) consume_half(b, 0);
                __syncthreads();
                if (whole) consume_half(b, 1);
            } else {
                if (i < t_count) {
                    if ((t_first + i + 1) * kTK <= Lk) consume(mode_c, mode_c, t_first + i, b);
                    else pend = i;
                }
            }
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
        }
        if (pend >= 0) consume(mode_c, mode_c, t_first + pend, pend & 1);
    };

    run_tiles(fixed_c);
    // Overflow vote: with m fixed at the first sub-tile's maximum - kPBias, a
    // later logit larger than that maximum by more than ~8 (log2) overflows
    // the rounded p to inf,
    // which makes this lane's row sum non-finite.  Any such row sends the
    // whole workgroup (it shares the LDS tiles) through the online path.
    {
        bool overflow = false;
#pragma unroll
        for (int j = 0; j < QB; ++j) {
            float l_check;
            if constexpr (G::kOnes) {
                constexpr int dd = D % 32;
                constexpr int rsel = 4 * (dd >> 3) + (dd & 3);
                l_check = acc[j][D / 32][rsel];
            } else {
                l_check = l_part[j];
            }
            overflow = overflow || !(__builtin_fabsf(l_check) < __builtin_inff());
        }
        // workgroup-wide OR through the (now idle) first LDS words
        int* vote = (int*)smem;
        const int wave_overflow = __any(overflow) ? 1 : 0;   // ballot with every lane active
        if (lane == 0) vote[wave] = wave_overflow;
        __syncthreads();
        int any = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) any |= vote[w];
        __syncthreads();
        if (any) {
            reset();
            run_tiles(online_c);
            // The merge below writes into the tile buffers; a wave of key
            // half 1 may still be reading its ragged last tile there (run_tiles
            // ends without a barrier after that tile).  The fixed-maximum pass
            // has the vote's barriers in between.
            __syncthreads();
        }
    }

    // ---- merge the key splits of every row (the block-merge rule): split s
    // > 0 leaves its O^T, m, max and l in LDS, split 0 folds them in
    constexpr int kMF = DN * 16 * 64 + 3 * 64;   // floats per query block
    auto mrg_of = [&](int s) { return (float*)smem + ((s - 1) * kQW + wq) * G::kMergeFloats; };
    if (kh != 0) {
        float* mrg = mrg_of(kh);
#pragma unroll
        for (int j = 0; j < QB; ++j) {
            float* mj = mrg + j * kMF;
#pragma unroll
            for (int n = 0; n < DN; ++n)
#pragma unroll
                for (int r = 0; r < 16; ++r) mj[(n * 16 + r) * 64 + lane] = acc[j][n][r];
            mj[DN * 16 * 64 + lane] = m_run[j];
            mj[DN * 16 * 64 + 64 + lane] = s_max[j];
            mj[DN * 16 * 64 + 128 + lane] = l_part[j];
        }
    }
    __syncthreads();
    if (kh != 0) return;
#pragma unroll
    for (int s = 1; s < G::kKS; ++s)
#pragma unroll
    for (int j = 0; j < QB; ++j) {
        const float* mj = mrg_of(s) + j * kMF;
        const float m_b = mj[DN * 16 * 64 + lane];
        const float m_new = fmaxf(m_run[j], m_b);
        const float a0 = fast_exp2(m_run[j] - m_new);   // exp2(-inf) = 0 for an empty split
        const float a1 = fast_exp2(m_b - m_new);
#pragma unroll
        for (int n = 0; n < DN; ++n)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[j][n][r] = acc[j][n][r] * a0 + mj[(n * 16 + r) * 64 + lane] * a1;
        s_max[j] = fmaxf(s_max[j], mj[DN * 16 * 64 + 64 + lane]);
        l_part[j] = l_part[j] * a0 + mj[DN * 16 * 64 + 128 + lane] * a1;
        m_run[j] = m_new;
    }

    // ---- epilogue: l, O / l, store
#pragma unroll
    for (int j = 0; j < QB; ++j) {
        float l;
        if constexpr (G::kOnes) {
            constexpr int dd = D % 32;               // position of the ones row in its d tile
            constexpr int hsel = (dd >> 2) & 1, rsel = 4 * (dd >> 3) + (dd & 3);
            const float own = acc[j][D / 32][rsel];
            const float other = half_partner(own, half);
            l = (half == hsel) ? own : other;
        } else {
            l = half_sum(l_part[j]);
        }
        const float inv = 1.0f / l;
        const int qrow = q0 + 32 * j + l32;
        if (qrow < Lq) {
            uint16_t* orow = OROWS ? out_base(O, bh, Lq, D, oh) + (size_t)qrow * out_stride(D, oh)
                                   : O + ((size_t)bh * Lq + qrow) * D;
#pragma unroll
            for (int n = 0; n < DN; ++n)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int d0 = 32 * n + 8 * g + 4 * half;
                    if (32 * n + 8 * g < D) {   // D % 8 == 0: then d0 + 3 < D for both halves
                        u32x2 w;
                        w[0] = pack2<ET>(acc[j][n][4 * g + 0] * inv, acc[j][n][4 * g + 1] * inv);
                        w[1] = pack2<ET>(acc[j][n][4 * g + 2] * inv, acc[j][n][4 * g + 3] * inv);
                        *(u32x2*)(orow + d0) = w;
                    }
                }
            if (LS && half == 0) {
                // Eq. 4 in natural units: L = max_j scale q.k, S = sum_j exp(scale q.k - L)
                float* o2 = LS + ((size_t)bh * Lq + qrow) * 2;
                o2[0] = s_max[j] * scale_abs;
                o2[1] = l * fast_exp2(m_run[j] - s_max[j] * c);
            }
        }
    }
}

template <int ET, int D, bool STATS, bool OROWS, int GEO>
hipError_t launch_kernel(const AttnArgs& a) {
    using G = Geom<D, GEO>;
    const int nqb = (a.Lq + G::kBQ - 1) / G::kBQ;
    const long long nblk = (long long)a.B * a.H * nqb;
    const float scale_abs = a.scale < 0 ? -a.scale : a.scale;
    const float c = scale_abs * kLog2e;
    auto kern = attn_fwd_lds_kernel<ET, D, STATS, OROWS, GEO>;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                                       G::kLdsBytes);
    if (attr != hipSuccess) return attr;
    hipLaunchKernelGGL(kern, dim3((unsigned)nblk), dim3(G::kThreads), G::kLdsBytes,
                       (hipStream_t)a.stream, (const uint16_t*)a.q, (const uint16_t*)a.k,
                       (const uint16_t*)a.v, (uint16_t*)a.out, a.ls, a.Lq, a.Lk, scale_abs, c,
                       a.scale < 0 ? 1 : 0, nqb, a.o_rows ? a.H : 0);
    return hipGetLastError();
}

template <int ET, int D>
hipError_t launch_d(const AttnArgs& a) {
    if constexpr (!Geom<D, kGeoNormal>::kFits || !Geom<D, kGeoSmall>::kFits) {
        return launch_attn_fwd_generic(a);
    } else {
        if (a.ls && a.o_rows) return hipErrorInvalidValue;   // no caller asks for both
        // tile copies address a head's K and V with 32-bit byte offsets
        if ((long long)a.Lk * D * 2 > 0x7fffffffLL) return launch_attn_fwd_generic(a);
        if (a.ls) return launch_kernel<ET, D, true, false, kGeoNormal>(a);
        // the geometry with the largest workgroups whose grid still covers the
        // 256 CUs (the smallest one when none does)
        const long long heads = (long long)a.B * a.H;
        const bool small = heads * ((a.Lq + 127) / 128) < 256;
        bool big = false;
        if constexpr (Geom<D, kGeoBig>::kFits) big = heads * ((a.Lq + 255) / 256) >= 256;
        if (small) {
            // keys split four ways (two waves per SIMD) once every split has
            // at least two tiles
            if constexpr (Geom<D, kGeoQuarter>::kFits) {
                if (a.Lk >= kQuarterMinKeys)
                    return a.o_rows ? launch_kernel<ET, D, false, true, kGeoQuarter>(a)
                                    : launch_kernel<ET, D, false, false, kGeoQuarter>(a);
            }
            return a.o_rows ? launch_kernel<ET, D, false, true, kGeoSmall>(a)
                            : launch_kernel<ET, D, false, false, kGeoSmall>(a);
        }
        if constexpr (Geom<D, kGeoBig>::kFits) {
            if (big) return a.o_rows ? launch_kernel<ET, D, false, true, kGeoBig>(a)
                                     : launch_kernel<ET, D, false, false, kGeoBig>(a);
        }
        return a.o_rows ? launch_kernel<ET, D, false, true, kGeoNormal>(a)
                        : launch_kernel<ET, D, false, false, kGeoNormal>(a);
    }
}

template <int ET, int... Ds>
hipError_t dispatch_d(const AttnArgs& a, std::integer_sequence<int, Ds...>) {
    hipError_t r = hipErrorInvalidValue;
    bool hit = ((a.D == 8 * (Ds + 1) ? (r = launch_d<ET, 8 * (Ds + 1)>(a), true) : false) || ...);
    return hit ? r : hipErrorInvalidValue;
}

}  // namespace

}  // namespace sdattn
