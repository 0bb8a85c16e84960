// sdattn_api.hip -- the C ABI of include/sdattn.h: argument checks, then one
// kernel launch on the caller's stream.  Every check runs before any HIP call,
// so a rejected call touches neither the device nor the outputs.
#include <math.h>
#include <stdint.h>

#include <climits>
#include <mutex>

#include "launch.h"
#include "sdattn.h"

// The static scratch of sdattn_attention_block_static: Q, K, V and O of one
// block between its launches, for callers that cannot allocate.  Each GPU the
// library runs on holds its own copy until the process ends.  In host code
// `scratch` names a host-side stand-in, never the device memory: its device
// address comes from hipGetSymbolAddress, once per device (scratch_address).
static __device__ __align__(256) char scratch[SDATTN_STATIC_SCRATCH_BYTES];

namespace {

thread_local int g_last_hip_error = 0;

bool aligned(const void* p, uintptr_t n) { return ((uintptr_t)p % n) == 0; }

// [p, p + n) and [q, q + m) share a byte
bool overlap(const void* p, unsigned long long n, const void* q, unsigned long long m) {
    const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + m && b < a + n;
}

// product of positive factors, or -1 when it reaches 2^62
long long checked_mul(std::initializer_list<long long> fs) {
    long long r = 1;
    for (long long f : fs) {
        if (f <= 0) return -1;
        if (r > (1LL << 62) / f) return -1;
        r *= f;
    }
    return r < (1LL << 62) ? r : -1;
}

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// The current device's address of `scratch`, looked up on the first call on
// that device (with it current) and kept: no allocation, no launch.
int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return SDATTN_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxScratchDevices) return SDATTN_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            g_last_hip_error = (int)(e != hipSuccess ? e : hipErrorInvalidSymbol);
            return SDATTN_ERR_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return SDATTN_OK;
}

int finish(hipError_t e) {
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return SDATTN_ERR_HIP;
    }
    return SDATTN_OK;
}

int check_attention(const void* q, const void* k, const void* v, const void* out, const float* ls,
                    int B, int H, int Lq, int Lk, int D, float scale, int dtype) {
    if (!q || !k || !v || !out) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || D < 1) return SDATTN_ERR_INVALID_ARG;
    if (!isfinite(scale)) return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16) {
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    }
    if (D % 8 != 0 || D > 256) return SDATTN_ERR_UNSUPPORTED;
    const long long nq = checked_mul({B, H, Lq, D});
    const long long nk = checked_mul({B, H, Lk, D});
    if (nq < 0 || nk < 0) return SDATTN_ERR_UNSUPPORTED;
    if (sdattn::attn_fwd_grid(B, H, Lq) > INT_MAX) return SDATTN_ERR_UNSUPPORTED;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16))
        return SDATTN_ERR_MISALIGNED;
    if (ls && !aligned(ls, 8)) return SDATTN_ERR_MISALIGNED;
    const unsigned long long qb = 2ULL * nq, kb = 2ULL * nk;
    if (overlap(out, qb, q, qb) || overlap(out, qb, k, kb) || overlap(out, qb, v, kb))
        return SDATTN_ERR_INVALID_ARG;
    if (ls) {
        const unsigned long long lb = 8ULL * (unsigned long long)(nq / D);
        if (overlap(ls, lb, q, qb) || overlap(ls, lb, k, kb) || overlap(ls, lb, v, kb) ||
            overlap(ls, lb, out, qb))
            return SDATTN_ERR_INVALID_ARG;
    }
    return SDATTN_OK;
}

int run_attention(const void* q, const void* k, const void* v, void* out, float* ls, int B, int H,
                  int Lq, int Lk, int D, float scale, int dtype, void* stream) {
    const int st = check_attention(q, k, v, out, ls, B, H, Lq, Lk, D, scale, dtype);
    if (st != SDATTN_OK) return st;
    (void)hipGetLastError();   // start from a clean error state for this launch
    sdattn::AttnArgs a{q, k, v, out, ls, B, H, Lq, Lk, D, scale, dtype, stream};
    return finish(sdattn::launch_attn_fwd(a));
}

int elem_size(int dtype) {
    switch (dtype) {
        case SDATTN_F16:
        case SDATTN_BF16: return 2;
        case SDATTN_F32: return 4;
        default: return 0;
    }
}

// Shared checks of sdattn_logits and sdattn_softmax_pv: sizes, types, and the
// element counts of the [B,H,Lq,D], [B,H,Lk,D] and [B,H,Lq,Lk] tensors.
int check_twopass(int B, int H, int Lq, int Lk, int D, int dtype, int a_dtype, long long* nq,
                  long long* nk, long long* na) {
    if (B < 1 || H < 1 || Lq < 1 || Lk < 1 || D < 1) return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16) {
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    }
    if (elem_size(a_dtype) == 0) return SDATTN_ERR_INVALID_ARG;
    if (D % 8 != 0 || D > 256) return SDATTN_ERR_UNSUPPORTED;
    *nq = checked_mul({B, H, Lq, D});
    *nk = checked_mul({B, H, Lk, D});
    *na = checked_mul({B, H, Lq, Lk, elem_size(a_dtype)});
    if (*nq < 0 || *nk < 0 || *na < 0) return SDATTN_ERR_UNSUPPORTED;
    if (sdattn::logits_grid(B, H, Lq, Lk) > INT_MAX || sdattn::attn_fwd_grid(B, H, Lq) > INT_MAX)
        return SDATTN_ERR_UNSUPPORTED;
    return SDATTN_OK;
}

// Checks of sdattn_linear; fills the launch arguments.
int check_linear(const void* x, const void* w, const void* bias, void* y, int B, int L, int K,
                 int N, int H, int x_layout, int y_layout, int dtype, void* stream,
                 sdattn::LinearArgs* args) {
    if (!x || !w || !y) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || L < 1 || K < 1 || N < 1) return SDATTN_ERR_INVALID_ARG;
    if ((x_layout != SDATTN_ROWS && x_layout != SDATTN_HEADS) ||
        (y_layout != SDATTN_ROWS && y_layout != SDATTN_HEADS))
        return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16) {
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    }
    const bool xh = x_layout == SDATTN_HEADS, yh = y_layout == SDATTN_HEADS;
    if ((xh || yh) && H < 1) return SDATTN_ERR_INVALID_ARG;
    if (K % 8 != 0 || N % 8 != 0 || K > 65536 || N > 65536) return SDATTN_ERR_UNSUPPORTED;
    if (xh && (K % H != 0 || (K / H) % 8 != 0)) return SDATTN_ERR_UNSUPPORTED;
    if (yh && (N % H != 0 || (N / H) % 8 != 0)) return SDATTN_ERR_UNSUPPORTED;
    const long long nx = checked_mul({B, L, K}), ny = checked_mul({B, L, N}), nw = checked_mul({N, K});
    if (nx < 0 || ny < 0 || nw < 0 || (long long)B * L > INT_MAX / 2) return SDATTN_ERR_UNSUPPORTED;
    if (sdattn::linear_grid(B, L, N) > INT_MAX) return SDATTN_ERR_UNSUPPORTED;
    if (!aligned(x, 16) || !aligned(w, 16) || !aligned(y, 16) || (bias && !aligned(bias, 8)))
        return SDATTN_ERR_MISALIGNED;
    const unsigned long long yb = 2ULL * ny;
    if (overlap(y, yb, x, 2ULL * nx) || overlap(y, yb, w, 2ULL * nw) ||
        (bias && overlap(y, yb, bias, 2ULL * N)))
        return SDATTN_ERR_INVALID_ARG;
    *args = sdattn::LinearArgs{x, w, bias, y, B, L, K, N, xh || yh ? H : 1, xh, yh, dtype, stream};
    return SDATTN_OK;
}

// Q, K, V (heads layout) and O (heads merged), each rounded up to 256 bytes
long long block_part(long long elems) { return (2 * elems + 255) / 256 * 256; }

}  // namespace

extern "C" {

int sdattn_forward(const void* q, const void* k, const void* v, void* out, int B, int H, int Lq,
                   int Lk, int D, float scale, void* stream) {
    return run_attention(q, k, v, out, nullptr, B, H, Lq, Lk, D, scale, SDATTN_F16, stream);
}

int sdattn_forward_ex(const void* q, const void* k, const void* v, void* out, float* ls, int B,
                      int H, int Lq, int Lk, int D, float scale, sdattn_dtype dtype, void* stream) {
    return run_attention(q, k, v, out, ls, B, H, Lq, Lk, D, scale, (int)dtype, stream);
}

int sdattn_softmax_rows(const void* a, float* ls, void* p, long long rows, long long cols,
                        float scale, sdattn_dtype dtype, void* stream) {
    if (!a || !ls) return SDATTN_ERR_INVALID_ARG;
    if (rows < 1 || cols < 1) return SDATTN_ERR_INVALID_ARG;
    if (!isfinite(scale)) return SDATTN_ERR_INVALID_ARG;
    int esize;
    switch (dtype) {
        case SDATTN_F16:
        case SDATTN_BF16: esize = 2; break;
        case SDATTN_F32: esize = 4; break;
        default: return SDATTN_ERR_INVALID_ARG;
    }
    const long long n = checked_mul({rows, cols, esize});
    if (n < 0) return SDATTN_ERR_UNSUPPORTED;
    if (!aligned(a, 16) || (p && !aligned(p, 16)) || !aligned(ls, 8)) return SDATTN_ERR_MISALIGNED;
    const unsigned long long lb = 8ULL * (unsigned long long)rows;
    if (overlap(ls, lb, a, n)) return SDATTN_ERR_INVALID_ARG;
    if (p && (overlap(p, n, a, n) || overlap(p, n, ls, lb))) return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    sdattn::SoftmaxArgs args{a, ls, p, rows, cols, scale, (int)dtype, stream};
    return finish(sdattn::launch_softmax_rows(args));
}

int sdattn_logits(const void* q, const void* k, void* a, int B, int H, int Lq, int Lk, int D,
                  float scale, sdattn_dtype dtype, sdattn_dtype a_dtype, void* stream) {
    if (!q || !k || !a) return SDATTN_ERR_INVALID_ARG;
    if (!isfinite(scale)) return SDATTN_ERR_INVALID_ARG;
    long long nq, nk, na;
    const int st = check_twopass(B, H, Lq, Lk, D, (int)dtype, (int)a_dtype, &nq, &nk, &na);
    if (st != SDATTN_OK) return st;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(a, 16)) return SDATTN_ERR_MISALIGNED;
    if (overlap(a, na, q, 2ULL * nq) || overlap(a, na, k, 2ULL * nk)) return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    sdattn::LogitsArgs args{q, k, a, B, H, Lq, Lk, D, scale, (int)dtype, (int)a_dtype, stream};
    return finish(sdattn::launch_logits(args));
}

int sdattn_softmax_pv(const void* a, const float* ls, const void* v, void* out, int B, int H,
                      int Lq, int Lk, int D, sdattn_dtype a_dtype, sdattn_dtype dtype, void* stream) {
    if (!a || !ls || !v || !out) return SDATTN_ERR_INVALID_ARG;
    long long nq, nk, na;
    const int st = check_twopass(B, H, Lq, Lk, D, (int)dtype, (int)a_dtype, &nq, &nk, &na);
    if (st != SDATTN_OK) return st;
    if (!aligned(a, 16) || !aligned(v, 16) || !aligned(out, 16) || !aligned(ls, 8))
        return SDATTN_ERR_MISALIGNED;
    const unsigned long long ob = 2ULL * nq, lb = 8ULL * (unsigned long long)(nq / D);
    if (overlap(out, ob, a, na) || overlap(out, ob, ls, lb) || overlap(out, ob, v, 2ULL * nk))
        return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    sdattn::SoftmaxPvArgs args{a, ls, v, out, B, H, Lq, Lk, D, (int)dtype, (int)a_dtype, stream};
    return finish(sdattn::launch_softmax_pv(args));
}

int sdattn_linear(const void* x, const void* w, const void* bias, void* y, int B, int L, int K,
                  int N, int H, sdattn_layout x_layout, sdattn_layout y_layout, sdattn_dtype dtype,
                  void* stream) {
    sdattn::LinearArgs args;
    const int st = check_linear(x, w, bias, y, B, L, K, N, H, (int)x_layout, (int)y_layout,
                                (int)dtype, stream, &args);
    if (st != SDATTN_OK) return st;
    (void)hipGetLastError();
    return finish(sdattn::launch_linear(args));
}

long long sdattn_attention_block_workspace(int B, int Lq, int Lk, int C) {
    // Lk == 0: Q and O only (sdattn_attention_block_kv)
    const long long nq = checked_mul({B, Lq, C}), nk = Lk == 0 ? 0 : checked_mul({B, Lk, C});
    if (nq < 0 || nk < 0) return -1;
    return 2 * block_part(nq) + 2 * block_part(nk);
}

int sdattn_attention_block(const void* x, const void* ctx, const void* wq, const void* wk,
                           const void* wv, const void* wo, const void* bo, void* out,
                           void* workspace, long long workspace_bytes, int B, int Lq, int Lk,
                           int C, int Cc, int H, float scale, sdattn_dtype dtype, void* stream) {
    if (!x || !ctx || !wq || !wk || !wv || !wo || !out || !workspace) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || Lq < 1 || Lk < 1 || C < 1 || Cc < 1 || H < 1) return SDATTN_ERR_INVALID_ARG;
    if (C % H != 0) return SDATTN_ERR_INVALID_ARG;
    const long long need = sdattn_attention_block_workspace(B, Lq, Lk, C);
    if (need < 0) return SDATTN_ERR_UNSUPPORTED;
    if (workspace_bytes < need) return SDATTN_ERR_INVALID_ARG;
    if (!aligned(workspace, 16)) return SDATTN_ERR_MISALIGNED;
    const int D = C / H;
    char* ws = (char*)workspace;
    void* q = ws;
    void* k = ws + block_part((long long)B * Lq * C);
    void* v = (char*)k + block_part((long long)B * Lk * C);
    void* o = (char*)v + block_part((long long)B * Lk * C);
    // the inputs and the output must stay clear of the workspace and of each other
    const unsigned long long ob = 2ULL * B * Lq * C;
    const void* ins[] = {x, ctx, wq, wk, wv, wo, bo};
    const unsigned long long insz[] = {2ULL * B * Lq * C, 2ULL * B * Lk * Cc, 2ULL * C * C,
                                       2ULL * C * Cc, 2ULL * C * Cc, 2ULL * C * C, 2ULL * C};
    for (int i = 0; i < 7; ++i) {
        if (!ins[i]) continue;
        if (overlap(ins[i], insz[i], workspace, (unsigned long long)need) ||
            overlap(ins[i], insz[i], out, ob))
            return SDATTN_ERR_INVALID_ARG;
    }
    if (overlap(out, ob, workspace, (unsigned long long)need)) return SDATTN_ERR_INVALID_ARG;
    sdattn::LinearArgs pq, pk, pv, po;
    int st;
    if ((st = check_linear(x, wq, nullptr, q, B, Lq, C, C, H, SDATTN_ROWS, SDATTN_HEADS, (int)dtype,
                           stream, &pq)) != SDATTN_OK ||
        (st = check_linear(ctx, wk, nullptr, k, B, Lk, Cc, C, H, SDATTN_ROWS, SDATTN_HEADS,
                           (int)dtype, stream, &pk)) != SDATTN_OK ||
        (st = check_linear(ctx, wv, nullptr, v, B, Lk, Cc, C, H, SDATTN_ROWS, SDATTN_HEADS,
                           (int)dtype, stream, &pv)) != SDATTN_OK ||
        (st = check_linear(o, wo, bo, out, B, Lq, C, C, H, SDATTN_ROWS, SDATTN_ROWS, (int)dtype,
                           stream, &po)) != SDATTN_OK)
        return st;
    if ((st = check_attention(q, k, v, o, nullptr, B, H, Lq, Lk, D, scale, (int)dtype)) != SDATTN_OK)
        return st;
    (void)hipGetLastError();
    hipError_t e;
    const sdattn::LinearArgs qkv[3] = {pq, pk, pv};
    if ((e = sdattn::launch_linear_group(qkv, 3)) != hipSuccess) return finish(e);
    // O leaves the attention with the heads merged ([B, Lq, C]), as the output
    // projection reads it
    sdattn::AttnArgs aa{q, k, v, o, nullptr, B, H, Lq, Lk, D, scale, (int)dtype, stream, 1};
    if ((e = sdattn::launch_attn_fwd(aa)) != hipSuccess) return finish(e);
    return finish(sdattn::launch_linear(po));
}

int sdattn_attention_block_static(const void* x, const void* ctx, const void* wq, const void* wk,
                                  const void* wv, const void* wo, const void* bo, void* out, int B,
                                  int Lq, int Lk, int C, int Cc, int H, float scale,
                                  sdattn_dtype dtype, void* stream) {
    // what needs no device address first: a refused size makes no HIP call
    if (!x || !ctx || !wq || !wk || !wv || !wo || !out) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || Lq < 1 || Lk < 1 || C < 1 || Cc < 1 || H < 1) return SDATTN_ERR_INVALID_ARG;
    if (C % H != 0) return SDATTN_ERR_INVALID_ARG;
    const long long need = sdattn_attention_block_workspace(B, Lq, Lk, C);
    if (need < 0) return SDATTN_ERR_UNSUPPORTED;
    if (need > SDATTN_STATIC_SCRATCH_BYTES) return SDATTN_ERR_SCRATCH;
    void* ws = nullptr;
    const int st = scratch_address(&ws);
    if (st != SDATTN_OK) return st;
    return sdattn_attention_block(x, ctx, wq, wk, wv, wo, bo, out, ws, SDATTN_STATIC_SCRATCH_BYTES, B, Lq,
                                  Lk, C, Cc, H, scale, dtype, stream);
}

int sdattn_project_kv(const void* ctx, const void* wk, const void* wv, void* k, void* v, int B,
                      int Lk, int Cc, int C, int H, sdattn_dtype dtype, void* stream) {
    if (!ctx || !wk || !wv || !k || !v) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || Lk < 1 || C < 1 || Cc < 1 || H < 1 || C % H != 0) return SDATTN_ERR_INVALID_ARG;
    sdattn::LinearArgs kv[2];
    int st;
    if ((st = check_linear(ctx, wk, nullptr, k, B, Lk, Cc, C, H, SDATTN_ROWS, SDATTN_HEADS,
                           (int)dtype, stream, &kv[0])) != SDATTN_OK ||
        (st = check_linear(ctx, wv, nullptr, v, B, Lk, Cc, C, H, SDATTN_ROWS, SDATTN_HEADS,
                           (int)dtype, stream, &kv[1])) != SDATTN_OK)
        return st;
    const unsigned long long kb = 2ULL * B * Lk * C;
    if (overlap(k, kb, v, kb) || overlap(k, kb, wv, 2ULL * C * Cc) ||
        overlap(v, kb, wk, 2ULL * C * Cc))
        return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    return finish(sdattn::launch_linear_group(kv, 2));
}

int sdattn_attention_block_kv(const void* x, const void* wq, const void* k, const void* v,
                              const void* wo, const void* bo, void* out, void* workspace,
                              long long workspace_bytes, int B, int Lq, int Lk, int C, int H,
                              float scale, sdattn_dtype dtype, void* stream) {
    if (!x || !wq || !k || !v || !wo || !out || !workspace) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || Lq < 1 || Lk < 1 || C < 1 || H < 1 || C % H != 0) return SDATTN_ERR_INVALID_ARG;
    const long long need = sdattn_attention_block_workspace(B, Lq, 0, C);
    if (need < 0) return SDATTN_ERR_UNSUPPORTED;
    if (workspace_bytes < need) return SDATTN_ERR_INVALID_ARG;
    if (!aligned(workspace, 16)) return SDATTN_ERR_MISALIGNED;
    const int D = C / H;
    void* q = workspace;
    void* o = (char*)workspace + block_part((long long)B * Lq * C);
    const unsigned long long ob = 2ULL * B * Lq * C;
    const void* ins[] = {x, wq, k, v, wo, bo};
    const unsigned long long insz[] = {2ULL * B * Lq * C, 2ULL * C * C, 2ULL * B * Lk * C,
                                       2ULL * B * Lk * C, 2ULL * C * C, 2ULL * C};
    for (int i = 0; i < 6; ++i) {
        if (!ins[i]) continue;
        if (overlap(ins[i], insz[i], workspace, (unsigned long long)need) ||
            overlap(ins[i], insz[i], out, ob))
            return SDATTN_ERR_INVALID_ARG;
    }
    if (overlap(out, ob, workspace, (unsigned long long)need)) return SDATTN_ERR_INVALID_ARG;
    sdattn::LinearArgs pq, po;
    int st;
    if ((st = check_linear(x, wq, nullptr, q, B, Lq, C, C, H, SDATTN_ROWS, SDATTN_HEADS, (int)dtype,
                           stream, &pq)) != SDATTN_OK ||
        (st = check_linear(o, wo, bo, out, B, Lq, C, C, H, SDATTN_ROWS, SDATTN_ROWS, (int)dtype,
                           stream, &po)) != SDATTN_OK)
        return st;
    if ((st = check_attention(q, k, v, o, nullptr, B, H, Lq, Lk, D, scale, (int)dtype)) != SDATTN_OK)
        return st;
    (void)hipGetLastError();
    hipError_t e;
    if ((e = sdattn::launch_linear(pq)) != hipSuccess) return finish(e);
    sdattn::AttnArgs aa{q, k, v, o, nullptr, B, H, Lq, Lk, D, scale, (int)dtype, stream, 1};
    if ((e = sdattn::launch_attn_fwd(aa)) != hipSuccess) return finish(e);
    return finish(sdattn::launch_linear(po));
}

int sdattn_group_norm(const void* x, const void* gamma, const void* beta, void* y, int B, int C,
                      long long HW, int G, float eps, sdattn_dtype dtype, void* stream) {
    if (!x || !y) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || C < 1 || HW < 1 || G < 1 || C % G != 0) return SDATTN_ERR_INVALID_ARG;
    if (!isfinite(eps) || eps < 0.0f) return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16)
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    const long long n = checked_mul({B, C, HW});
    if (n < 0 || (long long)B * G > INT_MAX) return SDATTN_ERR_UNSUPPORTED;
    if (!aligned(x, 16) || !aligned(y, 16) || (gamma && !aligned(gamma, 2)) ||
        (beta && !aligned(beta, 2)))
        return SDATTN_ERR_MISALIGNED;
    const unsigned long long nb = 2ULL * n;
    // y is x itself (in place) or disjoint from it; gamma and beta stay clear of y
    if (y != x && overlap(y, nb, x, nb)) return SDATTN_ERR_INVALID_ARG;
    if ((gamma && overlap(y, nb, gamma, 2ULL * C)) || (beta && overlap(y, nb, beta, 2ULL * C)))
        return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    sdattn::GroupNormArgs a{x, gamma, beta, y, B, C, HW, G, eps, (int)dtype, stream};
    return finish(sdattn::launch_group_norm(a));
}

int sdattn_geglu(const void* h, void* out, long long M, int F, sdattn_dtype dtype, void* stream) {
    if (!h || !out) return SDATTN_ERR_INVALID_ARG;
    if (M < 1 || F < 1) return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16)
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    if (F % 8 != 0) return SDATTN_ERR_UNSUPPORTED;
    const long long nh = checked_mul({M, 2LL * F});
    if (nh < 0) return SDATTN_ERR_UNSUPPORTED;
    if (!aligned(h, 16) || !aligned(out, 16)) return SDATTN_ERR_MISALIGNED;
    if (overlap(out, (unsigned long long)nh, h, 2ULL * nh)) return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    sdattn::GegluArgs a{h, out, M, F, (int)dtype, stream};
    return finish(sdattn::launch_geglu(a));
}

long long sdattn_winograd_weights_elems(int Co, int Ci) {
    const long long n = checked_mul({36, Co, Ci});
    return n < 0 ? -1 : n;
}

int sdattn_winograd_weights(const void* w, void* u, int Co, int Ci, sdattn_dtype dtype,
                            void* stream) {
    if (!w || !u) return SDATTN_ERR_INVALID_ARG;
    if (Co < 1 || Ci < 1) return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16)
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    const long long nu = sdattn_winograd_weights_elems(Co, Ci);
    if (nu < 0) return SDATTN_ERR_UNSUPPORTED;
    if (!aligned(w, 2) || !aligned(u, 16)) return SDATTN_ERR_MISALIGNED;
    if (overlap(u, 2ULL * nu, w, 2ULL * 9 * Co * Ci)) return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    sdattn::WinoFilterArgs a{w, u, Co, Ci, (int)dtype, stream};
    return finish(sdattn::launch_wino_filter(a));
}

// V [36][T][Ci] and M [36][T][Co], each rounded up to 256 bytes
long long sdattn_conv3x3_workspace(int B, int Ci, int Co, int H, int W) {
    if (B < 1 || Ci < 1 || Co < 1 || H < 1 || W < 1) return -1;
    const long long T = sdattn::wino_tiles(B, H, W);
    const long long nv = checked_mul({36, T, Ci}), nm = checked_mul({36, T, Co});
    if (nv < 0 || nm < 0) return -1;
    return block_part(nv) + block_part(nm);
}

int sdattn_conv3x3(const void* x, const void* u, const void* bias, void* y, void* workspace,
                   long long workspace_bytes, int B, int Ci, int Co, int H, int W,
                   sdattn_dtype dtype, void* stream) {
    if (!x || !u || !y || !workspace) return SDATTN_ERR_INVALID_ARG;
    if (B < 1 || Ci < 1 || Co < 1 || H < 1 || W < 1) return SDATTN_ERR_INVALID_ARG;
    if (dtype != SDATTN_F16 && dtype != SDATTN_BF16)
        return dtype == SDATTN_F32 ? SDATTN_ERR_UNSUPPORTED : SDATTN_ERR_INVALID_ARG;
    if (Ci % 8 != 0 || Co % 8 != 0 || Ci > 65536 || Co > 65536) return SDATTN_ERR_UNSUPPORTED;
    const long long nx = checked_mul({B, Ci, H, W}), ny = checked_mul({B, Co, H, W});
    const long long need = sdattn_conv3x3_workspace(B, Ci, Co, H, W);
    const long long T = sdattn::wino_tiles(B, H, W);
    // the input transform addresses 64 channel planes of one image in 32 bits
    if (nx < 0 || ny < 0 || need < 0 || T > INT_MAX / 2 || (long long)H * W > (1LL << 25) ||
        (long long)B * ((H + 3) / 4) * ((W + 31) / 32) > INT_MAX)
        return SDATTN_ERR_UNSUPPORTED;
    if (workspace_bytes < need) return SDATTN_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(u, 16) || !aligned(y, 16) || !aligned(workspace, 16) ||
        (bias && !aligned(bias, 2)))
        return SDATTN_ERR_MISALIGNED;
    const unsigned long long yb = 2ULL * ny, ub = 2ULL * 36 * Co * Ci, wb = (unsigned long long)need;
    if (overlap(y, yb, x, 2ULL * nx) || overlap(y, yb, u, ub) || overlap(y, yb, workspace, wb) ||
        (bias && overlap(y, yb, bias, 2ULL * Co)) || overlap(workspace, wb, x, 2ULL * nx) ||
        overlap(workspace, wb, u, ub) || (bias && overlap(workspace, wb, bias, 2ULL * Co)))
        return SDATTN_ERR_INVALID_ARG;
    (void)hipGetLastError();
    void* m = (char*)workspace + block_part(36 * T * Ci);
    sdattn::WinoConvArgs a{x, u, bias, y, workspace, m, B, Ci, Co, H, W, (int)dtype, stream};
    return finish(sdattn::launch_wino_conv(a));
}

const char* sdattn_status_str(int status) {
    switch (status) {
        case SDATTN_OK: return "ok";
        case SDATTN_ERR_INVALID_ARG: return "invalid argument";
        case SDATTN_ERR_UNSUPPORTED: return "unsupported size or type";
        case SDATTN_ERR_MISALIGNED: return "misaligned pointer";
        case SDATTN_ERR_HIP: return "HIP runtime error";
        case SDATTN_ERR_SCRATCH: return "needs more than the static scratch holds";
        default: return "unknown status";
    }
}

int sdattn_last_hip_error(void) { return g_last_hip_error; }

const char* sdattn_version(void) { return "sdattn 0.1.0 (gfx950)"; }

}  // extern "C"
