// Host side of the C ABI declared in include/dfa.h: argument validation,
// dispatch of the plan codes to the HIP kernels, the seeded plan generator
// and the per-thread error message.
//
// Validation always runs before the first HIP call, so every argument error
// is reported on a machine without a GPU.
#include "dfa.h"

#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include <string>
#include <vector>

#include "dfa_internal.h"

namespace {

thread_local std::string g_last_error;

void vrecord(const char* fmt, va_list ap) {
    char buf[512];
    vsnprintf(buf, sizeof buf, fmt, ap);
    g_last_error = buf;
}

dfa_status fail(dfa_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vrecord(fmt, ap);
    va_end(ap);
    return st;
}

dfa_status hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return DFA_OK;
    return fail(DFA_ERR_HIP, "%s: %s (%s)", what, hipGetErrorName(e), hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// [a, a + na) and [b, b + nb) intersect
bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

bool overlaps(const void* a, const void* b, size_t n) { return overlaps(a, n, b, n); }

struct Shape {
    int B, H, L, d, w;
    size_t bytes;    // one [B,H,L,d] bf16 tensor
    size_t rbytes;   // the fp32 residual [B,H,L,d]
};

dfa_status check_shape(int B, int H, int L, int d, int w, Shape* s) {
    if (B <= 0 || H <= 0 || L <= 0 || d <= 0)
        return fail(DFA_ERR_INVALID_ARG, "sizes must be positive (B=%d H=%d L=%d d=%d)", B, H, L, d);
    if (w < 0) return fail(DFA_ERR_INVALID_ARG, "window half-width w=%d must be >= 0", w);
    // token indexes (plus a tile) are int arithmetic in the kernels
    if (L > (1 << 30)) return fail(DFA_ERR_INVALID_ARG, "L=%d is too large (at most 2^30 tokens)", L);
    const unsigned long long elems = (unsigned long long)B * H * L * d;
    if (elems > (1ULL << 40)) return fail(DFA_ERR_INVALID_ARG, "tensor of %llu elements is too large", elems);
    if ((unsigned long long)B * H > (1ULL << 24)) return fail(DFA_ERR_INVALID_ARG, "B*H=%lld is too large", (long long)B * H);
    if (!dfa::head_dim_supported(d)) return fail(DFA_ERR_UNSUPPORTED, "head dim d=%d is not built (supported: 64, 72)", d);
    s->B = B;
    s->H = H;
    s->L = L;
    s->d = d;
    s->w = w;
    s->bytes = (size_t)elems * 2;
    s->rbytes = (size_t)elems * 4;
    return DFA_OK;
}

dfa_status check_ptr(const void* p, const char* name) {
    if (!p) return fail(DFA_ERR_INVALID_ARG, "%s is NULL", name);
    if (!aligned16(p)) return fail(DFA_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return DFA_OK;
}

dfa_status check_qkv(const void* Q, const void* K, const void* V) {
    dfa_status st;
    if ((st = check_ptr(Q, "Q")) != DFA_OK) return st;
    if ((st = check_ptr(K, "K")) != DFA_OK) return st;
    return check_ptr(V, "V");
}

// an output buffer of out_bytes must not overlap any input tensor of in_bytes
dfa_status check_out_vs_inputs(const void* out, const char* name, const void* Q, const void* K, const void* V,
                               size_t in_bytes, size_t out_bytes) {
    if (overlaps(out, out_bytes, Q, in_bytes) || overlaps(out, out_bytes, K, in_bytes) ||
        overlaps(out, out_bytes, V, in_bytes))
        return fail(DFA_ERR_INVALID_ARG, "%s overlaps Q, K or V", name);
    return DFA_OK;
}

dfa_status check_out_vs_inputs(const void* out, const char* name, const void* Q, const void* K, const void* V,
                               size_t bytes) {
    return check_out_vs_inputs(out, name, Q, K, V, bytes, bytes);
}

dfa::AttnLaunch make_launch(const void* Q, const void* K, const void* V, const Shape& s) {
    dfa::AttnLaunch a{};
    a.Q = Q;
    a.K = K;
    a.V = V;
    a.B = s.B;
    a.H = s.H;
    a.L = s.L;
    a.d = s.d;
    a.w = s.w;
    return a;
}

// The output cache is written by computed steps unless it is O itself.
bool cache_is_separate(const void* O, const void* Oc) { return Oc != nullptr && Oc != O; }

dfa_status check_cache(const void* O, const void* Oc, const void* Q, const void* K, const void* V, const void* R,
                       size_t bytes, size_t rbytes) {
    if (!cache_is_separate(O, Oc)) return DFA_OK;
    dfa_status st;
    if ((st = check_ptr(Oc, "Ocache")) != DFA_OK) return st;
    if ((st = check_out_vs_inputs(Oc, "Ocache", Q, K, V, bytes)) != DFA_OK) return st;
    if (overlaps(Oc, O, bytes)) return fail(DFA_ERR_INVALID_ARG, "Ocache partially overlaps O");
    if (R && overlaps(Oc, bytes, R, rbytes)) return fail(DFA_ERR_INVALID_ARG, "Ocache overlaps R");
    return DFA_OK;
}

}  // namespace

int dfa::set_error(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vrecord(fmt, ap);
    va_end(ap);
    return status;
}

extern "C" {

const char* dfa_last_error(void) { return g_last_error.c_str(); }

const char* dfa_version(void) { return "0.6.0"; }

dfa_status dfa_attn_full(const void* Q, const void* K, const void* V, void* O, void* R, int B, int H, int L, int d,
                         int w, hipStream_t stream) {
    (void)R;
    Shape s;
    dfa_status st;
    if ((st = check_shape(B, H, L, d, w, &s)) != DFA_OK) return st;
    if ((st = check_qkv(Q, K, V)) != DFA_OK) return st;
    if ((st = check_ptr(O, "O")) != DFA_OK) return st;
    if ((st = check_out_vs_inputs(O, "O", Q, K, V, s.bytes)) != DFA_OK) return st;
    dfa::AttnLaunch a = make_launch(Q, K, V, s);
    a.dst[0] = O;
    a.ndst = 1;
    return hip_status(dfa::attn_full(a, stream), "dfa_attn_full launch");
}

dfa_status dfa_attn_full_and_residual(const void* Q, const void* K, const void* V, void* O, void* R, int B, int H,
                                      int L, int d, int w, hipStream_t stream) {
    Shape s;
    dfa_status st;
    if ((st = check_shape(B, H, L, d, w, &s)) != DFA_OK) return st;
    if ((st = check_qkv(Q, K, V)) != DFA_OK) return st;
    if ((st = check_ptr(O, "O")) != DFA_OK) return st;
    if ((st = check_ptr(R, "R")) != DFA_OK) return st;
    if ((st = check_out_vs_inputs(O, "O", Q, K, V, s.bytes)) != DFA_OK) return st;
    if ((st = check_out_vs_inputs(R, "R", Q, K, V, s.bytes, s.rbytes)) != DFA_OK) return st;
    if (overlaps(O, s.bytes, R, s.rbytes)) return fail(DFA_ERR_INVALID_ARG, "O and R overlap");
    dfa::AttnLaunch a = make_launch(Q, K, V, s);
    a.dst[0] = O;
    a.ndst = 1;
    a.Rout = R;
    return hip_status(dfa::attn_refresh(a, stream), "dfa_attn_full_and_residual launch");
}

dfa_status dfa_attn_window_plus_residual(const void* Q, const void* K, const void* V, void* O, const void* R, int B,
                                         int H, int L, int d, int w, hipStream_t stream) {
    Shape s;
    dfa_status st;
    if ((st = check_shape(B, H, L, d, w, &s)) != DFA_OK) return st;
    if ((st = check_qkv(Q, K, V)) != DFA_OK) return st;
    if ((st = check_ptr(O, "O")) != DFA_OK) return st;
    if (R && !aligned16(R)) return fail(DFA_ERR_INVALID_ARG, "R is not 16-byte aligned");
    if ((st = check_out_vs_inputs(O, "O", Q, K, V, s.bytes)) != DFA_OK) return st;
    if (R && overlaps(O, s.bytes, R, s.rbytes)) return fail(DFA_ERR_INVALID_ARG, "O and R overlap");
    dfa::AttnLaunch a = make_launch(Q, K, V, s);
    a.dst[0] = O;
    a.ndst = 1;
    a.Rin = R;
    return hip_status(dfa::attn_window(a, stream), "dfa_attn_window_plus_residual launch");
}

dfa_status dfa_plan_step(int code, const void* Q, const void* K, const void* V, void* O, void* R, void* Ocache,
                         int B, int H, int L, int d, int w, hipStream_t stream) {
    if (code < DFA_FULL || code > DFA_WARS_ASC_REUSE) return fail(DFA_ERR_INVALID_ARG, "unknown plan code %d", code);
    Shape s;
    dfa_status st;
    if ((st = check_shape(B, H, L, d, w, &s)) != DFA_OK) return st;
    if ((st = check_ptr(O, "O")) != DFA_OK) return st;
    const bool sep = cache_is_separate(O, Ocache);

    if (code == DFA_AST_REUSE) {
        // no attention: Q/K/V are not read and may be NULL
        if (!Ocache) return fail(DFA_ERR_INVALID_ARG, "AST needs the layer's output cache (Ocache is NULL)");
        if (!sep) return DFA_OK;  // the output already lives in the cache
        if ((st = check_ptr(Ocache, "Ocache")) != DFA_OK) return st;
        if (overlaps(O, Ocache, s.bytes)) return fail(DFA_ERR_INVALID_ARG, "Ocache partially overlaps O");
        return hip_status(dfa::launch_copy(Ocache, O, s.bytes, stream), "AST copy launch");
    }

    const bool half_batch = code == DFA_ASC_REUSE || code == DFA_WARS_ASC_REFRESH || code == DFA_WARS_ASC_REUSE;
    if (half_batch && (B % 2)) return fail(DFA_ERR_INVALID_ARG, "plan code %d needs an even batch (B=%d)", code, B);
    if ((st = check_qkv(Q, K, V)) != DFA_OK) return st;
    if ((st = check_out_vs_inputs(O, "O", Q, K, V, s.bytes)) != DFA_OK) return st;
    const bool uses_r = code == DFA_WARS_REFRESH || code == DFA_WARS_REUSE || code == DFA_WARS_ASC_REFRESH ||
                        code == DFA_WARS_ASC_REUSE;
    if (uses_r) {
        if ((st = check_ptr(R, "R")) != DFA_OK) return st;
        if ((st = check_out_vs_inputs(R, "R", Q, K, V, s.bytes, s.rbytes)) != DFA_OK) return st;
        if (overlaps(O, s.bytes, R, s.rbytes)) return fail(DFA_ERR_INVALID_ARG, "O and R overlap");
    }
    if ((st = check_cache(O, Ocache, Q, K, V, uses_r ? R : nullptr, s.bytes, s.rbytes)) != DFA_OK) return st;

    dfa::AttnLaunch a = make_launch(Q, K, V, s);
    a.dst[0] = O;
    a.ndst = 1;
    if (half_batch) {
        // attention on the conditional half (entries 0..B/2-1, which are also
        // the first half of R); every output tile is also stored at its
        // unconditional partner (and in the cache)
        const size_t half = s.bytes / 2;
        a.B = B / 2;
        a.dst[a.ndst++] = (char*)O + half;
        if (sep) {
            a.dst[a.ndst++] = Ocache;
            a.dst[a.ndst++] = (char*)Ocache + half;
        }
    } else if (sep) {
        a.dst[a.ndst++] = Ocache;
    }
    switch (code) {
        case DFA_FULL:
            return hip_status(dfa::attn_full(a, stream), "FULL launch");
        case DFA_ASC_REUSE:
            return hip_status(dfa::attn_asc(a, stream), "ASC launch");
        case DFA_WARS_REFRESH:
        case DFA_WARS_ASC_REFRESH:
            a.Rout = R;
            return hip_status(dfa::attn_refresh(a, stream), "WA-RS refresh launch");
        default:  // DFA_WARS_REUSE, DFA_WARS_ASC_REUSE
            a.Rin = R;
            return hip_status(dfa::attn_window(a, stream), "WA-RS reuse launch");
    }
}

// ---------------------------------------------------------------------------
// The attention module: projections and one module step
// ---------------------------------------------------------------------------
namespace {

struct Region {
    const void* p;
    size_t n;
    const char* name;
};

// every output region must avoid every input region and every other output
dfa_status check_regions(const Region* outs, int nout, const Region* ins, int nin) {
    for (int i = 0; i < nout; ++i) {
        if (!outs[i].p) continue;
        for (int j = 0; j < nin; ++j)
            if (ins[j].p && overlaps(outs[i].p, outs[i].n, ins[j].p, ins[j].n))
                return fail(DFA_ERR_INVALID_ARG, "%s overlaps %s", outs[i].name, ins[j].name);
        for (int j = i + 1; j < nout; ++j)
            if (outs[j].p && overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n))
                return fail(DFA_ERR_INVALID_ARG, "%s overlaps %s", outs[i].name, outs[j].name);
    }
    return DFA_OK;
}

dfa_status check_proj_shape(int B, int H, int L, int d, Shape* s) {
    dfa_status st;
    if ((st = check_shape(B, H, L, d, 0, s)) != DFA_OK) return st;
    // the projections index the B * L tokens with int arithmetic
    if ((long long)B * L > (1LL << 30))
        return fail(DFA_ERR_INVALID_ARG, "B*L=%lld tokens is too large for a projection (at most 2^30)", (long long)B * L);
    if (!dfa::proj_shape_supported(H, d))
        return fail(DFA_ERR_UNSUPPORTED, "projection width H*d=%d is not a multiple of 128 (H=%d d=%d)", H * d, H, d);
    return DFA_OK;
}

dfa_status check_bias(const void* b, const char* name) {
    if (b && !aligned16(b)) return fail(DFA_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return DFA_OK;
}

}  // namespace

dfa_status dfa_qkv_proj(const void* X, const void* Wqkv, const void* bqkv, void* Q, void* K, void* V, int B, int H,
                        int L, int d, hipStream_t stream) {
    Shape s;
    dfa_status st;
    if ((st = check_proj_shape(B, H, L, d, &s)) != DFA_OK) return st;
    if ((st = check_ptr(X, "X")) != DFA_OK) return st;
    if ((st = check_ptr(Wqkv, "Wqkv")) != DFA_OK) return st;
    if ((st = check_bias(bqkv, "bqkv")) != DFA_OK) return st;
    if ((st = check_qkv(Q, K, V)) != DFA_OK) return st;
    const size_t C = (size_t)H * d;
    const Region outs[] = {{Q, s.bytes, "Q"}, {K, s.bytes, "K"}, {V, s.bytes, "V"}};
    const Region ins[] = {{X, s.bytes, "X"}, {Wqkv, 3 * C * C * 2, "Wqkv"}, {bqkv, 3 * C * 4, "bqkv"}};
    if ((st = check_regions(outs, 3, ins, 3)) != DFA_OK) return st;
    dfa::ProjLaunch a{};
    a.W = Wqkv;
    a.act = X;
    a.bias = bqkv;
    a.dst[0] = Q;
    a.dst[1] = K;
    a.dst[2] = V;
    a.ndst = 3;
    a.B = B;
    a.H = H;
    a.L = L;
    a.d = d;
    return hip_status(dfa::launch_qkv_proj(a, stream), "QKV projection launch");
}

dfa_status dfa_out_proj(const void* O, const void* Wo, const void* bo, void* Y, int B, int H, int L, int d,
                        hipStream_t stream) {
    Shape s;
    dfa_status st;
    if ((st = check_proj_shape(B, H, L, d, &s)) != DFA_OK) return st;
    if ((st = check_ptr(O, "O")) != DFA_OK) return st;
    if ((st = check_ptr(Wo, "Wo")) != DFA_OK) return st;
    if ((st = check_bias(bo, "bo")) != DFA_OK) return st;
    if ((st = check_ptr(Y, "Y")) != DFA_OK) return st;
    const size_t C = (size_t)H * d;
    const Region outs[] = {{Y, s.bytes, "Y"}};
    const Region ins[] = {{O, s.bytes, "O"}, {Wo, C * C * 2, "Wo"}, {bo, C * 4, "bo"}};
    if ((st = check_regions(outs, 1, ins, 3)) != DFA_OK) return st;
    dfa::ProjLaunch a{};
    a.W = Wo;
    a.act = O;
    a.bias = bo;
    a.dst[0] = Y;
    a.ndst = 1;
    a.B = B;
    a.H = H;
    a.L = L;
    a.d = d;
    return hip_status(dfa::launch_out_proj(a, stream), "output projection launch");
}

dfa_status dfa_module_step(int code, const void* X, const void* Wqkv, const void* bqkv, const void* Wo, const void* bo,
                           void* Q, void* K, void* V, void* O, void* R, void* Y, void* Ycache, int B, int H, int L,
                           int d, int w, hipStream_t stream) {
    if (code < DFA_FULL || code > DFA_WARS_ASC_REUSE) return fail(DFA_ERR_INVALID_ARG, "unknown plan code %d", code);
    Shape s;
    dfa_status st;
    if ((st = check_proj_shape(B, H, L, d, &s)) != DFA_OK) return st;
    if (w < 0) return fail(DFA_ERR_INVALID_ARG, "window half-width w=%d must be >= 0", w);
    s.w = w;
    if ((st = check_ptr(Y, "Y")) != DFA_OK) return st;
    const bool sep = cache_is_separate(Y, Ycache);

    if (code == DFA_AST_REUSE) {
        // the whole module is skipped: only the cached module output is read
        if (!Ycache) return fail(DFA_ERR_INVALID_ARG, "AST needs the module's output cache (Ycache is NULL)");
        if (!sep) return DFA_OK;
        if ((st = check_ptr(Ycache, "Ycache")) != DFA_OK) return st;
        if (overlaps(Y, Ycache, s.bytes)) return fail(DFA_ERR_INVALID_ARG, "Ycache partially overlaps Y");
        return hip_status(dfa::launch_copy(Ycache, Y, s.bytes, stream), "AST copy launch");
    }

    const bool half_batch = code == DFA_ASC_REUSE || code == DFA_WARS_ASC_REFRESH || code == DFA_WARS_ASC_REUSE;
    if (half_batch && (B % 2)) return fail(DFA_ERR_INVALID_ARG, "plan code %d needs an even batch (B=%d)", code, B);
    const bool uses_r = code == DFA_WARS_REFRESH || code == DFA_WARS_REUSE || code == DFA_WARS_ASC_REFRESH ||
                        code == DFA_WARS_ASC_REUSE;
    if ((st = check_ptr(X, "X")) != DFA_OK) return st;
    if ((st = check_ptr(Wqkv, "Wqkv")) != DFA_OK) return st;
    if ((st = check_ptr(Wo, "Wo")) != DFA_OK) return st;
    if ((st = check_bias(bqkv, "bqkv")) != DFA_OK) return st;
    if ((st = check_bias(bo, "bo")) != DFA_OK) return st;
    if ((st = check_qkv(Q, K, V)) != DFA_OK) return st;
    if ((st = check_ptr(O, "O")) != DFA_OK) return st;
    if (uses_r && (st = check_ptr(R, "R")) != DFA_OK) return st;
    if (sep && (st = check_ptr(Ycache, "Ycache")) != DFA_OK) return st;
    const size_t C = (size_t)H * d;
    const Region outs[] = {{Q, s.bytes, "Q"},
                           {K, s.bytes, "K"},
                           {V, s.bytes, "V"},
                           {O, s.bytes, "O"},
                           {uses_r ? R : nullptr, s.rbytes, "R"},
                           {Y, s.bytes, "Y"},
                           {sep ? Ycache : nullptr, s.bytes, "Ycache"}};
    const Region ins[] = {{X, s.bytes, "X"},
                          {Wqkv, 3 * C * C * 2, "Wqkv"},
                          {bqkv, 3 * C * 4, "bqkv"},
                          {Wo, C * C * 2, "Wo"},
                          {bo, C * 4, "bo"}};
    if ((st = check_regions(outs, 7, ins, 5)) != DFA_OK) return st;

    const int Bc = half_batch ? B / 2 : B;
    const size_t half = s.bytes / 2;
    dfa::ProjLaunch pq{};
    pq.W = Wqkv;
    pq.act = X;
    pq.bias = bqkv;
    pq.dst[0] = Q;
    pq.dst[1] = K;
    pq.dst[2] = V;
    pq.ndst = 3;
    pq.B = Bc;
    pq.H = H;
    pq.L = L;
    pq.d = d;
    if ((st = hip_status(dfa::launch_qkv_proj(pq, stream), "QKV projection launch")) != DFA_OK) return st;

    dfa::AttnLaunch a = make_launch(Q, K, V, s);
    a.B = Bc;
    a.dst[0] = O;
    a.ndst = 1;
    hipError_t e;
    switch (code) {
        case DFA_FULL:
        case DFA_ASC_REUSE:
            e = dfa::attn_full(a, stream);
            break;
        case DFA_WARS_REFRESH:
        case DFA_WARS_ASC_REFRESH:
            a.Rout = R;
            e = dfa::attn_refresh(a, stream);
            break;
        default:  // DFA_WARS_REUSE, DFA_WARS_ASC_REUSE
            a.Rin = R;
            e = dfa::attn_window(a, stream);
            break;
    }
    if ((st = hip_status(e, "module attention launch")) != DFA_OK) return st;

    dfa::ProjLaunch po{};
    po.W = Wo;
    po.act = O;
    po.bias = bo;
    po.dst[po.ndst++] = Y;
    if (half_batch) po.dst[po.ndst++] = (char*)Y + half;
    if (sep) {
        po.dst[po.ndst++] = Ycache;
        if (half_batch) po.dst[po.ndst++] = (char*)Ycache + half;
    }
    po.B = Bc;
    po.H = H;
    po.L = L;
    po.d = d;
    return hip_status(dfa::launch_out_proj(po, stream), "output projection launch");
}

// ---------------------------------------------------------------------------
// Seeded plan generator
// ---------------------------------------------------------------------------
namespace {

// SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): a Weyl sequence with the golden-ratio increment
// followed by two xor-shift-multiply rounds.
struct SplitMix64 {
    uint64_t x;
    uint64_t next() {
        x += 0x9E3779B97F4A7C15ULL;
        uint64_t z = x;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
        return z ^ (z >> 31);
    }
};

}  // namespace

dfa_status dfa_plan_make(uint64_t seed, int n_layers, int n_steps, int refresh_every, int B, int32_t* code,
                         int32_t* r_src, int32_t* o_src) {
    if (n_layers <= 0 || n_steps <= 0 || B <= 0 || refresh_every < 0)
        return fail(DFA_ERR_INVALID_ARG, "bad plan dimensions (layers=%d steps=%d refresh_every=%d B=%d)", n_layers,
                    n_steps, refresh_every, B);
    if ((long long)n_layers * n_steps > (1LL << 30)) return fail(DFA_ERR_INVALID_ARG, "plan too large");
    if (!code || !r_src || !o_src) return fail(DFA_ERR_INVALID_ARG, "plan output arrays must not be NULL");

    SplitMix64 rng{seed};
    std::vector<int> last_refresh(n_layers, -1);  // step of the layer's latest REFRESH
    std::vector<int> cached(n_layers, -1);        // step whose output the layer's cache holds
    for (int t = 0; t < n_steps; ++t) {
        for (int l = 0; l < n_layers; ++l) {
            const uint64_t hi = rng.next() >> 32;
            int c = (int)((hi * 5u) >> 32);
            if (c == DFA_AST_REUSE && cached[l] < 0) c = DFA_FULL;
            if (c == DFA_WARS_REFRESH || c == DFA_WARS_REUSE) {
                if (refresh_every > 0) {
                    const bool stale = last_refresh[l] < 0 || t - last_refresh[l] >= refresh_every;
                    c = stale ? DFA_WARS_REFRESH : DFA_WARS_REUSE;
                } else if (c == DFA_WARS_REUSE && last_refresh[l] < 0) {
                    c = DFA_WARS_REFRESH;
                }
            }
            if (c == DFA_ASC_REUSE && (B & 1))
                return fail(DFA_ERR_INVALID_ARG, "ASC drawn at step %d layer %d with odd B=%d", t, l, B);
            const size_t e = (size_t)t * n_layers + l;
            code[e] = c;
            r_src[e] = (c == DFA_WARS_REUSE) ? last_refresh[l] : -1;
            if (c == DFA_AST_REUSE) {
                o_src[e] = cached[l];
            } else {
                o_src[e] = t;
                cached[l] = t;
            }
            if (c == DFA_WARS_REFRESH) last_refresh[l] = t;
        }
    }
    return DFA_OK;
}

}  // extern "C"
