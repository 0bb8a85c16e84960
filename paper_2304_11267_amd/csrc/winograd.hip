// winograd.hip -- the 3x3 convolutions (stride 1, zero padding 1) of Sec. 3.3
// by Winograd's minimal filtering algorithm F(4x4, 3x3), the tile size the
// paper selects (Table 2: 4x fewer products, 2.25x the input tensor, 4x the
// weights).
//
// For one 4x4 output tile Y of one output channel, with the 6x6 input patch d
// of every input channel c and the 3x3 kernels g:
//   Y = A^T [ sum_c (G g_c G^T) .* (B^T d_c B) ] A
// with the 6-point transforms below (interpolation points 0, 1, -1, 1/2, -2
// and infinity: against the common 0, +-1, +-2 they make the transformed
// input smaller -- |V| at most 57 instead of 270 for unit inputs -- and the
// fp16 result about 2.5x closer to the exact convolution, measured on UNet
// shapes).  The sum over input channels at each of the 36 positions xi of
// the 6x6 transformed tile is a matrix product, so the convolution becomes:
//   1. U[xi][o][c] = (G g_oc G^T)[xi]     once per layer (weights are fixed)
//   2. V[xi][t][c] = (B^T d_tc B)[xi]     input transform, t = tile
//   3. M[xi] = V[xi] U[xi]^T              36 products [T x Ci] x [Ci x Co] on
//                                          the matrix cores (linear.hip, batched)
//   4. y = A^T M[.][t][o] A + bias        output transform
// U, V and M are stored in the input type (fp16/bf16) with fp32 arithmetic
// inside each step.  Feature maps are channel-major [B, C, H, W]; tiles run
// over ceil(H/4) x ceil(W/4) per image, the partial tiles at the right and
// bottom edges reading zeros and writing only the pixels inside the map.
#include "device.h"
#include "launch.h"

namespace sdattn {

namespace {

// The transforms (derived from the interpolation points above; B^T is 6x6,
// G is 6x3, A^T is 4x6).
__device__ constexpr float kBT[6][6] = {{1, -1.5f, -2, 1.5f, 1, 0},   {0, -1, 0.5f, 2.5f, 1, 0},
                                        {0, 1, -2.5f, 0.5f, 1, 0},    {0, -2, -1, 2, 1, 0},
                                        {0, 0.5f, -1, -0.5f, 1, 0},   {0, 1, -1.5f, -2, 1.5f, 1}};
__device__ constexpr float kG[6][3] = {{1, 0, 0},
                                       {1.0f / 3, 1.0f / 3, 1.0f / 3},
                                       {-1.0f / 3, 1.0f / 3, -1.0f / 3},
                                       {-16.0f / 15, -8.0f / 15, -4.0f / 15},
                                       {1.0f / 15, -2.0f / 15, 4.0f / 15},
                                       {0, 0, 1}};
__device__ constexpr float kAT[4][6] = {{1, 1, 1, 1, 1, 0},
                                        {0, 1, -1, 0.5f, -2, 0},
                                        {0, 1, 1, 0.25f, 4, 0},
                                        {0, 1, -1, 0.125f, -8, 1}};

// input transform: 8 tiles of a tile row x 64 channels per workgroup (the V
// stores of a tile are then whole 128-byte lines)
constexpr int kInTiles = 8;
constexpr int kInChan = 64;
constexpr int kPatchCols = 4 * kInTiles + 8;   // input columns staged: 4*tx0 - 4 .. 4*tx0 + 35
constexpr int kPlane = 6 * kPatchCols + 8;     // halves per channel plane in LDS (padded)
// output transform: 16 tiles (64 pixels, whole output rows of 128 bytes) x 32
// channels, one (tile, channel) per thread; the staged output rows are
// [row][channel][68 halves], so that 32 consecutive channels land in 32
// different LDS banks (a channel-major [channel][row][64] staging put them
// all in one bank: 30x the bank-conflict cycles, 7.2 instead of 5.2 us at the
// 64x64 level)
constexpr int kTilesPerWg = 16;
constexpr int kChanPerWg = 32;
constexpr int kOutThreads = kTilesPerWg * kChanPerWg;
constexpr int kOutRow = 4 * kTilesPerWg + 4;

// 1. U[xi][o][c] = (G g G^T)[xi], one thread per (o, c).
template <int ET>
__global__ __launch_bounds__(256) void wino_filter_kernel(const uint16_t* __restrict__ Wt,
                                                          uint16_t* __restrict__ U, int Co, int Ci) {
    const long long q = (long long)blockIdx.x * 256 + threadIdx.x;
    if (q >= (long long)Co * Ci) return;
    const uint16_t* g9 = Wt + q * 9;   // w[o][c][3][3], q = o*Ci + c
    float g[3][3];
#pragma unroll
    for (int i = 0; i < 9; ++i) g[i / 3][i % 3] = to_float<ET>(g9[i]);
    float t[6][3];
#pragma unroll
    for (int i = 0; i < 6; ++i)
#pragma unroll
        for (int c = 0; c < 3; ++c) t[i][c] = kG[i][0] * g[0][c] + kG[i][1] * g[1][c] + kG[i][2] * g[2][c];
    const size_t stride = (size_t)Co * Ci;
#pragma unroll
    for (int i = 0; i < 6; ++i)
#pragma unroll
        for (int j = 0; j < 6; ++j)
            U[(6 * i + j) * stride + q] =
                from_float<ET>(t[i][0] * kG[j][0] + t[i][1] * kG[j][1] + t[i][2] * kG[j][2]);
}

// 2. V[xi][t][c] = (B^T d B)[xi].  A workgroup takes 8 tiles of one tile row
// and 64 channels: the 6 x 40 input window of each channel goes to LDS (8-byte
// loads when W % 4 == 0), then each thread transforms the patches of one tile
// in two consecutive channels and writes 36 channel pairs, consecutive lanes
// on consecutive pairs.
template <int ET>
__global__ __launch_bounds__(256) void wino_input_kernel(const uint16_t* __restrict__ X,
                                                         uint16_t* __restrict__ V, int Ci, int H,
                                                         int W, int th, int tw, int nseg, int T) {
    __shared__ uint16_t patch[kInChan * kPlane];
    const int cb = blockIdx.y * kInChan;
    const int seg = blockIdx.x % nseg;
    const int brow = blockIdx.x / nseg;        // b * th + ty
    const int b = brow / th, ty = brow - b * th;
    const int tx0 = seg * kInTiles;
    const int r0 = 4 * ty - 1, c0 = 4 * tx0 - 4;
    const int tid = threadIdx.x;

    // this workgroup's channel planes; offsets inside them fit in 32 bits
    const uint16_t* xb = X + ((size_t)b * Ci + cb) * H * W;
    const int nch = min(kInChan, Ci - cb);
    if (W % 4 == 0) {
        // 32 channels x 6 rows x 18 chunks of 4 columns: every load issued
        // before the first LDS write, so their latencies overlap
        constexpr int kRowChunks = kPatchCols / 4;
        constexpr int kChunks = kInChan * 6 * kRowChunks;
        constexpr int kPer = (kChunks + 255) / 256;
        u32x2 v[kPer];
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int q = tid + 256 * i;
            const int row = q / kRowChunks, k = q - row * kRowChunks;   // row = ch * 6 + r
            const int ch = row / 6, r = row - ch * 6;
            const int gr = r0 + r, gc = c0 + 4 * k;
            const bool in = q < kChunks && ch < nch && (unsigned)gr < (unsigned)H &&
                            (unsigned)gc < (unsigned)W;
            v[i] = in ? *(const u32x2*)(xb + (unsigned)((ch * H + gr) * W + gc)) : u32x2{0u, 0u};
        }
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
            const int q = tid + 256 * i;
            const int row = q / kRowChunks, k = q - row * kRowChunks;
            if (q < kChunks) *(u32x2*)(patch + (row / 6) * kPlane + (row % 6) * kPatchCols + 4 * k) = v[i];
        }
    } else {
#pragma unroll 1
        for (int q = tid; q < kInChan * 6 * kPatchCols; q += 256) {
            const int row = q / kPatchCols, cc = q - row * kPatchCols;
            const int ch = row / 6, r = row - ch * 6;
            const int gr = r0 + r, gc = c0 + cc;
            const bool in = ch < nch && (unsigned)gr < (unsigned)H && (unsigned)gc < (unsigned)W;
            patch[ch * kPlane + r * kPatchCols + cc] = in ? xb[(unsigned)((ch * H + gr) * W + gc)] : (uint16_t)0;
        }
    }
    __syncthreads();

    // one tile and two consecutive channels per thread (Ci % 8 == 0, so both
    // exist together): 4-byte stores of the channel pair
    static_assert(kInTiles * kInChan / 2 == 256, "one (tile, channel pair) per thread");
    {
        const int cp = tid % (kInChan / 2), t = tid / (kInChan / 2);
        const int ch = 2 * cp;
        if (tx0 + t < tw && cb + ch < Ci) {
            const uint16_t* src = patch + ch * kPlane + 4 * t + 3;   // global column 4*(tx0 + t) - 1
            float d0[6][6], d1[6][6];
#pragma unroll
            for (int i = 0; i < 6; ++i)
#pragma unroll
                for (int j = 0; j < 6; ++j) {
                    d0[i][j] = to_float<ET>(src[i * kPatchCols + j]);
                    d1[i][j] = to_float<ET>(src[kPlane + i * kPatchCols + j]);
                }
            const size_t tg = (size_t)brow * tw + tx0 + t;   // tile index (b*th + ty)*tw + tx
            const size_t stride = (size_t)T * Ci;
            uint16_t* vo = V + tg * Ci + cb + ch;
            // one row of B^T d at a time, then that row of (B^T d) B
#pragma unroll
            for (int i = 0; i < 6; ++i) {
                float s0[6], s1[6];
#pragma unroll
                for (int j = 0; j < 6; ++j) {
                    float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
                    for (int r = 0; r < 6; ++r)
                        if (kBT[i][r] != 0.0f) {
                            a0 += kBT[i][r] * d0[r][j];
                            a1 += kBT[i][r] * d1[r][j];
                        }
                    s0[j] = a0;
                    s1[j] = a1;
                }
#pragma unroll
                for (int j = 0; j < 6; ++j) {
                    float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
                    for (int r = 0; r < 6; ++r)
                        if (kBT[j][r] != 0.0f) {
                            a0 += s0[r] * kBT[j][r];
                            a1 += s1[r] * kBT[j][r];
                        }
                    *(uint32_t*)(vo + (6 * i + j) * stride) = pack2<ET>(a0, a1);
                }
            }
        }
    }
}

// 4. y = A^T M A + bias.  A workgroup takes 16 tiles of one tile row and 32
// output channels; each thread transforms one tile of one output channel
// into LDS, then the 4 x 64 output window of each channel is written row by
// row.
template <int ET>
__global__ __launch_bounds__(kOutThreads) void wino_output_kernel(const uint16_t* __restrict__ Mt,
                                                                  const uint16_t* __restrict__ Bias,
                                                                  uint16_t* __restrict__ Y, int Co, int H,
                                                                  int W, int th, int tw, int nseg, int T) {
    __shared__ __attribute__((aligned(16))) uint16_t out[4 * kChanPerWg * kOutRow];
    const int ob = blockIdx.y * kChanPerWg;
    const int seg = blockIdx.x % nseg;
    const int brow = blockIdx.x / nseg;
    const int b = brow / th, ty = brow - b * th;
    const int tx0 = seg * kTilesPerWg;
    const int tid = threadIdx.x;

    {
        const int ch = tid % kChanPerWg, t = tid / kChanPerWg;
        if (tx0 + t < tw && ob + ch < Co) {
            const size_t tg = (size_t)brow * tw + tx0 + t;
            const size_t stride = (size_t)T * Co;
            const uint16_t* mi = Mt + tg * Co + ob + ch;
            float m[6][6];
#pragma unroll
            for (int i = 0; i < 6; ++i)
#pragma unroll
                for (int j = 0; j < 6; ++j) m[i][j] = to_float<ET>(mi[(6 * i + j) * stride]);
            const float bias = Bias ? to_float<ET>(Bias[ob + ch]) : 0.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float s[6];   // row i of A^T m
#pragma unroll
                for (int j = 0; j < 6; ++j) {
                    float a = 0.0f;
#pragma unroll
                    for (int r = 0; r < 6; ++r)
                        if (kAT[i][r] != 0.0f) a += kAT[i][r] * m[r][j];
                    s[j] = a;
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    float a = bias;
#pragma unroll
                    for (int r = 0; r < 6; ++r)
                        if (kAT[j][r] != 0.0f) a += s[r] * kAT[j][r];
                    out[(i * kChanPerWg + ch) * kOutRow + 4 * t + j] = from_float<ET>(a);
                }
            }
        }
    }
    __syncthreads();

    // rows 4*ty .. 4*ty + 3, columns 4*tx0 .. 4*tx0 + 63 of each channel
    const int cbase = 4 * tx0;
    if (W % 4 == 0) {
        for (int q = tid; q < kChanPerWg * 4 * 16; q += kOutThreads) {
            const int ch = q / 64, rem = q - ch * 64;
            const int r = rem / 16, k = rem - r * 16;
            const int gr = 4 * ty + r, gc = cbase + 4 * k;
            if (ob + ch < Co && gr < H && gc < W)
                *(u32x2*)(Y + (((size_t)b * Co + ob + ch) * H + gr) * W + gc) =
                    *(const u32x2*)(out + (r * kChanPerWg + ch) * kOutRow + 4 * k);
        }
    } else {
        for (int q = tid; q < kChanPerWg * 4 * 64; q += kOutThreads) {
            const int ch = q / 256, rem = q - ch * 256;
            const int r = rem / 64, cc = rem - r * 64;
            const int gr = 4 * ty + r, gc = cbase + cc;
            if (ob + ch < Co && gr < H && gc < W)
                Y[(((size_t)b * Co + ob + ch) * H + gr) * W + gc] = out[(r * kChanPerWg + ch) * kOutRow + cc];
        }
    }
}

template <int ET>
hipError_t launch_filter_e(const WinoFilterArgs& a) {
    const long long n = (long long)a.Co * a.Ci;
    hipLaunchKernelGGL(wino_filter_kernel<ET>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       (hipStream_t)a.stream, (const uint16_t*)a.w, (uint16_t*)a.u, a.Co, a.Ci);
    return hipGetLastError();
}

template <int ET>
hipError_t launch_conv_e(const WinoConvArgs& a) {
    const int th = (a.H + 3) / 4, tw = (a.W + 3) / 4;
    const int nseg = (tw + kTilesPerWg - 1) / kTilesPerWg;
    const int nseg_in = (tw + kInTiles - 1) / kInTiles;
    const long long T = (long long)a.B * th * tw;
    uint16_t* V = (uint16_t*)a.v;
    uint16_t* M = (uint16_t*)a.m;
    hipStream_t s = (hipStream_t)a.stream;
    const dim3 gin((unsigned)(a.B * th * nseg_in), (unsigned)((a.Ci + kInChan - 1) / kInChan));
    hipLaunchKernelGGL(wino_input_kernel<ET>, gin, dim3(256), 0, s, (const uint16_t*)a.x, V, a.Ci,
                       a.H, a.W, th, tw, nseg_in, (int)T);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // 36 products M[xi] = V[xi] U[xi]^T: tiles are the rows, input channels the
    // reduced dimension, output channels the columns
    LinearArgs la{};
    la.x = V;
    la.w = a.u;
    la.bias = nullptr;
    la.y = M;
    la.B = 1;
    la.L = (int)T;
    la.K = a.Ci;
    la.N = a.Co;
    la.H = 1;
    la.x_heads = la.y_heads = false;
    la.dtype = ET;
    la.stream = a.stream;
    la.batch = 36;
    la.sx = T * a.Ci;
    la.sw = (long long)a.Co * a.Ci;
    la.sy = T * a.Co;
    if ((e = launch_linear(la)) != hipSuccess) return e;
    const dim3 gout((unsigned)(a.B * th * nseg), (unsigned)((a.Co + kChanPerWg - 1) / kChanPerWg));
    hipLaunchKernelGGL(wino_output_kernel<ET>, gout, dim3(kOutThreads), 0, s, (const uint16_t*)M,
                       (const uint16_t*)a.bias, (uint16_t*)a.y, a.Co, a.H, a.W, th, tw, nseg, (int)T);
    return hipGetLastError();
}

}  // namespace

long long wino_tiles(int B, int H, int W) { return (long long)B * ((H + 3) / 4) * ((W + 3) / 4); }

hipError_t launch_wino_filter(const WinoFilterArgs& a) {
    return a.dtype == kF16 ? launch_filter_e<kF16>(a) : launch_filter_e<kBF16>(a);
}

hipError_t launch_wino_conv(const WinoConvArgs& a) {
    return a.dtype == kF16 ? launch_conv_e<kF16>(a) : launch_conv_e<kBF16>(a);
}

}  // namespace sdattn
