// sdattn_api.hip -- the C ABI of include/sdattn.h: argument checks, then one
// kernel launch on the caller's stream.  Every check runs before any HIP call,
// so a rejected call touches neither the device nor the outputs.
#include <math.h>
#include <stdint.h>

#include <climits>

#include "launch.h"
#include "sdattn.h"

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

const char* sdattn_status_str(int status) {
    switch (status) {
        case SDATTN_OK: return "ok";
        case SDATTN_ERR_INVALID_ARG: return "invalid argument";
        case SDATTN_ERR_UNSUPPORTED: return "unsupported size or type";
        case SDATTN_ERR_MISALIGNED: return "misaligned pointer";
        case SDATTN_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

int sdattn_last_hip_error(void) { return g_last_hip_error; }

const char* sdattn_version(void) { return "sdattn 0.1.0 (gfx950)"; }

}  // extern "C"
