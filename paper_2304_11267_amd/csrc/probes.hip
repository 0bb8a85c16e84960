// probes.hip -- measurement kernels (libsdattn_probes.so, include/sdattn_probes.h).
//
// They compute nothing of the attention.  The benchmark runs them to report
// what the chip sustains beside its published peaks: the fp16 matrix-core
// rate and the shader clock under that load (near-constant and random
// operands), the v_exp_f32 and v_fma_f32 rates and whether each runs while
// the matrix core of the same SIMD is busy, the self-attention tile's
// instruction mix without its data movement, HBM streaming rates, and a plain
// copy with the cross-attention kernel's grid and byte pattern (the floor for
// a kernel that moves those bytes).
// Every loop is bounded by its arguments and every access is inside the
// caller's buffers.
#include "device.h"
#include "sdattn_probes.h"

namespace sdattn {
namespace {

// fp16 pairs of random sign and mantissa with magnitudes in [1/4, 2): operand
// bits that toggle like real activations (the matrix core's power, and so the
// clock it sustains, depends on them)
__device__ __forceinline__ uint32_t noise_h2(uint32_t i) {
    const uint32_t h = i * 2654435761u ^ (i >> 7) * 40503u;
    const uint32_t lo = (h & 0x83ffu) | (0x3400u + ((h >> 10) & 0x0c00u));
    const uint32_t g = h * 2246822519u;
    const uint32_t hi = (g & 0x83ffu) | (0x3400u + ((g >> 10) & 0x0c00u));
    return lo | (hi << 16);
}

// Four independent 32x32x16 f16 accumulators: back-to-back matrix-core work,
// on near-constant operands or (NOISE) on four random A and B operands taken
// in turn, so that the inputs of consecutive MFMAs differ.
template <bool NOISE>
__device__ __forceinline__ float mfma_stream(int iters) {
    f16x8 a[4], b[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (NOISE) {
                const uint32_t k = 64u * (uint32_t)(threadIdx.x * 4 + j) + 2u * (uint32_t)i;
                const uint32_t x = noise_h2(k), y = noise_h2(k + 1);
                a[j][2 * i] = __builtin_bit_cast(_Float16, (uint16_t)x);
                a[j][2 * i + 1] = __builtin_bit_cast(_Float16, (uint16_t)(x >> 16));
                b[j][2 * i] = __builtin_bit_cast(_Float16, (uint16_t)y);
                b[j][2 * i + 1] = __builtin_bit_cast(_Float16, (uint16_t)(y >> 16));
            } else {
                a[j][2 * i] = a[j][2 * i + 1] = (_Float16)((threadIdx.x & 63) * 0.001f);
                b[j][2 * i] = b[j][2 * i + 1] = (_Float16)0.5f;
            }
        }
    f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int it = 0; it < iters; ++it) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[0], b[0], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[NOISE ? 1 : 0], b[NOISE ? 1 : 0], c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[NOISE ? 2 : 0], b[NOISE ? 2 : 0], c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[NOISE ? 3 : 0], b[NOISE ? 3 : 0], c3, 0, 0, 0);
    }
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
    return s;
}

// 16 independent chains of one VALU operation: 0 = v_fma_f32, 1 = v_exp_f32.
template <int OP>
__device__ __forceinline__ float valu_stream(int iters) {
    float f[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) f[i] = 0.25f + 0.001f * (float)((threadIdx.x & 63) + i);
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            if constexpr (OP == 0) f[i] = fmaf(f[i], 0.999f, 0.0001f);
            else f[i] = __builtin_amdgcn_exp2f(-f[i]);   // stays in [0.5, 1]
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += f[i];
    return s;
}

// The self-attention tile's instruction mix without its data movement: per
// iteration two 32-query x 32-key pairs sharing every operand read, as the
// D = 40 kernel runs them -- K rows from LDS (three 16-byte reads) into 2 x 3
// chained 32x32x16 MFMAs, then per pair 16 FMAs (c s - m), 16 exponentials
// and 8 conversions, then V^T by transposing LDS reads into 2 x 4 MFMAs.
// The LDS tile is written once and only read; exps = 0 leaves out the
// exponentials.  Returns nothing but a checksum per lane.
__device__ __forceinline__ uint32_t pack_h2(float x, float y) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    const f2 v = {x, y};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
}

__device__ __forceinline__ f32x16 mm32(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                  0, 0, 0);
}

template <bool EXPS>
__device__ __forceinline__ void tile_softmax(const f32x16& st, float c, float m, u32x4 (&p)[2]) {
    float e[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) e[r] = fmaf(st[r], c, -m);
    if constexpr (EXPS) {
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(e[r]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int w = 0; w < 4; ++w) p[u][w] = pack_h2(e[8 * u + 2 * w], e[8 * u + 2 * w + 1]);
}


template <bool EXPS, bool NOISE>
__device__ float tile_mix(int iters, int stagger) {
    constexpr int D = 40;
    __shared__ __attribute__((aligned(16))) char lds[32 * 1024];
    for (int i = threadIdx.x; i < 32 * 1024 / 16; i += 512)
        *(u32x4*)(lds + 16 * i) = NOISE ? u32x4{noise_h2(4 * i), noise_h2(4 * i + 1), noise_h2(4 * i + 2), noise_h2(4 * i + 3)}
                                        : u32x4{0x2c002c00u, 0x3c00u, (uint32_t)i & 0x3ffu, 0x2c00u};
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l32 = lane & 31, half = lane >> 5;
    const char* base = lds + (wave & 3) * 8192;   // 64 keys of K (5 KiB), then V
    const int k_off = (l32 * D + 8 * half) * 2;
    const int g = lane >> 4, i16 = lane & 15;
    const int v_off = 64 * D * 2 + ((4 * (g >> 1) + (i16 >> 2)) * D + 16 * (g & 1) + 4 * (i16 & 3)) * 2;
    u32x4 q0[3], q1[3];
#pragma unroll
    for (int s = 0; s < 3; ++s) {
        if constexpr (NOISE) {
            const uint32_t b = 4096u * (uint32_t)(threadIdx.x * 3 + s);
            q0[s] = u32x4{noise_h2(b), noise_h2(b + 1), noise_h2(b + 2), noise_h2(b + 3)};
        } else {
            q0[s] = u32x4{0x3c003c00u + (uint32_t)lane, 0x3c00u, 0x3800u + (uint32_t)s, 0x3c00u};
        }
        q1[s] = q0[s] ^ 3u;
    }
    f32x16 acc[4] = {};
    const float c = 0.228f, m = NOISE ? 2.0f : 0.5f;
    // the second wave of each SIMD starts `stagger` x 64 cycles late
    if (wave >= 4)
        for (int z = 0; z < stagger; ++z) __builtin_amdgcn_s_sleep(1);
    for (int it = 0; it < iters; ++it) {
        const int sub = it & 1;
        f32x16 s0 = {}, s1 = {};
#pragma unroll
        for (int s = 0; s < 3; ++s) {
            const u32x4 a = *(const u32x4*)(base + k_off + (32 * sub * D + 16 * s) * 2);
            s0 = mm32(a, q0[s], s0);
            s1 = mm32(a, q1[s], s1);
        }
        u32x4 p0[2], p1[2];
        tile_softmax<EXPS>(s0, c, m, p0);
        tile_softmax<EXPS>(s1, c, m, p1);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int n = 0; n < 2; ++n) {
                const char* vb = base + v_off + (32 * sub + 16 * u) * D * 2 + n * 64;
                const u32x2 lo = lds_read_tr(vb);
                const u32x2 hi = lds_read_tr(vb + 8 * D * 2);
                const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                acc[n] = mm32(a, p0[u], acc[n]);
                acc[2 + n] = mm32(a, p1[u], acc[2 + n]);
            }
    }
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[0][r] + acc[1][r] + acc[2][r] + acc[3][r];
    return s;
}

__global__ __launch_bounds__(512, 2) void tile_kernel(float* __restrict__ out, int iters, int mode, int stagger,
                                                       unsigned long long* __restrict__ clk) {
    const bool first = blockIdx.x == 0 && threadIdx.x == 0;
    unsigned long long t0 = 0, r0 = 0;
    if (first) {
        t0 = __builtin_amdgcn_s_memtime();
        r0 = __builtin_amdgcn_s_memrealtime();
    }
    float s;
    switch (mode) {
        case 0: s = tile_mix<false, false>(iters, stagger); break;
        case 1: s = tile_mix<true, false>(iters, stagger); break;
        case 2: s = tile_mix<false, true>(iters, stagger); break;
        default: s = tile_mix<true, true>(iters, stagger); break;
    }
    out[(size_t)blockIdx.x * 512 + threadIdx.x] = s;
    if (first && clk) {
        const unsigned long long t1 = __builtin_amdgcn_s_memtime();
        const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
        clk[0] = t0;
        clk[1] = t1;
        clk[2] = r0;
        clk[3] = r1;
    }
}

__global__ __launch_bounds__(512) void mix_kernel(float* __restrict__ out, int mode, int it_m, int it_v,
                                                  unsigned long long* __restrict__ clk) {
    const int wave = threadIdx.x >> 6;
    const bool first = blockIdx.x == 0 && wave == 0;
    unsigned long long t0 = 0, r0 = 0;
    if (first) {
        t0 = __builtin_amdgcn_s_memtime();
        r0 = __builtin_amdgcn_s_memrealtime();
    }
    const bool low = wave < 4;   // waves 0-3: one per SIMD; 4-7: the second of each SIMD
    float s = 0.0f;
    switch (mode) {
        case 0: s = mfma_stream<false>(it_m); break;
        case 8: s = mfma_stream<true>(it_m); break;
        case 1: s = valu_stream<0>(it_v); break;
        case 2: s = valu_stream<1>(it_v); break;
        case 3: s = low ? mfma_stream<false>(it_m) : valu_stream<0>(it_v); break;
        case 4: s = low ? mfma_stream<false>(it_m) : valu_stream<1>(it_v); break;
        case 5: s = low ? mfma_stream<false>(it_m) : 0.0f; break;
        case 6: s = low ? 0.0f : valu_stream<0>(it_v); break;
        default: s = low ? 0.0f : valu_stream<1>(it_v); break;
    }
    out[(size_t)blockIdx.x * 512 + threadIdx.x] = s;
    if (first && clk && (threadIdx.x & 63) == 0) {
        const unsigned long long t1 = __builtin_amdgcn_s_memtime();
        const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
        clk[0] = t0;
        clk[1] = t1;
        clk[2] = r0;
        clk[3] = r1;
    }
}

__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                   long long n) {
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void read_kernel(const u32x4* __restrict__ src, long long n,
                                                   unsigned* __restrict__ sink) {
    const long long stride = (long long)gridDim.x * blockDim.x;
    u32x4 x = {0u, 0u, 0u, 0u};
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) x ^= src[i];
    sink[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = x[0] ^ x[1] ^ x[2] ^ x[3];
}

// W waves per workgroup (one 32-row strip each) of one head: the data
// movement of the short-sequence attention kernel without its arithmetic.  K and V (all Lk rows) and each wave's 32 query rows go
// global -> LDS with 16-byte direct copies, all issued before any wait; after
// the workgroup's barrier each wave stores its rows back out as O with
// 16-byte lanes, as the kernel's epilogue does.
__global__ __launch_bounds__(512) void strip_copy_kernel(const char* __restrict__ Q, const char* __restrict__ K,
                                                         const char* __restrict__ V, char* __restrict__ O,
                                                         unsigned* __restrict__ sink, int Lq, int Lk, int D,
                                                         int nqb, int kv_span, int W) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    const int bh = tile / nqb;
    const int qb = tile - bh * nqb;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int kv_bytes = Lk * D * 2;                 // <= kv_span, a multiple of 1024
    const char* kh = K + (size_t)bh * kv_bytes;
    const char* vh = V + (size_t)bh * kv_bytes;
    const int nkv = kv_span / 1024;
    for (int c = wave; c < 2 * nkv; c += W) {
        const bool isv = c >= nkv;
        const int cc = isv ? c - nkv : c;
        const int byte = cc * 1024 + lane * 16;
        if (byte < kv_bytes)
            __builtin_amdgcn_global_load_lds((isv ? vh : kh) + byte,
                                             (lds_void_t*)(smem + (isv ? kv_span : 0) + cc * 1024), 16, 0, 0);
    }
    const int strip = 32 * D * 2;
    const int q0 = qb * 32 * W + wave * 32;
    const int bytes = max(0, min(32, Lq - q0)) * D * 2;
    char* stage = smem + 2 * kv_span + wave * strip;
    const char* qs = Q + ((size_t)bh * Lq + max(q0, 0)) * D * 2;
    for (int c = 0; c * 1024 < bytes; ++c) {
        const int byte = c * 1024 + lane * 16;
        if (byte < bytes) __builtin_amdgcn_global_load_lds(qs + byte, (lds_void_t*)(stage + c * 1024), 16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    char* os = O + ((size_t)bh * Lq + max(q0, 0)) * D * 2;
    for (int b = lane * 16; b < bytes; b += 1024) *(u32x4*)(os + b) = *(const u32x4*)(stage + b);
    if (threadIdx.x == 0) sink[blockIdx.x] = *(const unsigned*)smem ^ *(const unsigned*)(smem + kv_span);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace
}  // namespace sdattn

using namespace sdattn;

extern "C" int sdattn_probe_mix(int mode, int blocks, int it_m, int it_v, float* out,
                                unsigned long long* clk, void* stream) {
    if (!out || mode < 0 || mode > 8 || blocks < 1 || blocks > 65536 || it_m < 0 || it_v < 0 ||
        it_m > (1 << 20) || it_v > (1 << 20))
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(mix_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream, out, mode, it_m, it_v, clk);
    return (int)hipGetLastError();
}

extern "C" int sdattn_probe_tile(int blocks, int iters, int mode, int stagger, float* out,
                                 unsigned long long* clk, void* stream) {
    if (!out || blocks < 1 || blocks > 65536 || iters < 1 || iters > (1 << 20) || mode < 0 || mode > 3 ||
        stagger < 0 || stagger > 64)
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(tile_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream, out, iters, mode, stagger, clk);
    return (int)hipGetLastError();
}

extern "C" int sdattn_probe_copy(const void* src, void* dst, long long bytes, int blocks, void* stream) {
    if (!src || !dst || bytes < 16 || bytes % 16 || blocks < 1 || blocks > (1 << 20) || !aligned16(src) ||
        !aligned16(dst))
        return (int)hipErrorInvalidValue;
    const char* s = (const char*)src;
    const char* d = (const char*)dst;
    if (s < d + bytes && d < s + bytes) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const u32x4*)src,
                       (u32x4*)dst, bytes / 16);
    return (int)hipGetLastError();
}

extern "C" int sdattn_probe_read(const void* src, long long bytes, unsigned* sink, int blocks, void* stream) {
    if (!src || !sink || bytes < 16 || bytes % 16 || blocks < 1 || blocks > (1 << 20) || !aligned16(src))
        return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(read_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const u32x4*)src,
                       bytes / 16, sink);
    return (int)hipGetLastError();
}

extern "C" int sdattn_probe_strip_copy(const void* q, const void* k, const void* v, void* o, unsigned* sink,
                                       int B, int H, int Lq, int Lk, int D, int waves, void* stream) {
    if (!q || !k || !v || !o || !sink || B < 1 || H < 1 || Lq < 1 || Lk < 1 || Lk > 128 || D < 8 || D > 160 ||
        D % 8 || (waves != 2 && waves != 4 && waves != 8) || !aligned16(q) || !aligned16(k) || !aligned16(v) ||
        !aligned16(o))
        return (int)hipErrorInvalidValue;
    const int nqb = (Lq + 32 * waves - 1) / (32 * waves);
    const long long nblk = (long long)B * H * nqb;
    if (nblk > (1 << 24)) return (int)hipErrorInvalidValue;
    const int kv_span = (Lk * D * 2 + 1023) / 1024 * 1024;
    const int lds = 2 * kv_span + waves * 32 * D * 2;   // <= 2 * 40 KiB + 80 KiB
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(strip_copy_kernel),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return (int)attr;
    hipLaunchKernelGGL(strip_copy_kernel, dim3((unsigned)nblk), dim3(64 * waves), lds, (hipStream_t)stream,
                       (const char*)q, (const char*)k, (const char*)v, (char*)o, sink, Lq, Lk, D, nqb, kv_span,
                       waves);
    return (int)hipGetLastError();
}
