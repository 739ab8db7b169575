// Host side of the plan search (Sec. 3.5, Alg. 1) and of the MRAE entry
// points: the greedy loop runs on the host and drives the library's own
// module steps, residual adds and loss reduction on the GPU.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "dfa.h"
#include "dfa_internal.h"

namespace {

constexpr size_t ALIGN = 256;
constexpr int MRAE_PARTIALS = 1024;

size_t round_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// Fraction of the uncompressed module's FLOPs that a strategy keeps (the
// module of Table 2: projections 8 L C^2 per batch entry, attention 4 C per
// (query, key) pair; the band is truncated at the sequence ends).
double kept_fraction(int code, long long L, long long C, long long w) {
    if (code == DFA_AST_REUSE) return 0.0;
    if (code == DFA_ASC_REUSE) return 0.5;
    const double band = w >= L - 1 ? (double)L * L : (double)(L * (2 * w + 1) - w * (w + 1));
    const double proj = 8.0 * L * C * C;
    const double wars = (proj + 4.0 * C * band) / (proj + 4.0 * C * (double)L * L);
    return code == DFA_WARS_REUSE ? wars : wars / 2;
}

struct Layout {
    size_t bytes, rbytes;   // one [B][L][C] bf16 tensor, one fp32 residual
    size_t q, k, v, o, yt, hc, ht, oref, rs, part, res, layers, per_layer, total;
};

Layout layout(int n_layers, int B, int H, int L, int d) {
    Layout s{};
    s.bytes = (size_t)B * L * H * d * 2;
    s.rbytes = s.bytes * 2;
    size_t off = 0;
    size_t* slots[] = {&s.q, &s.k, &s.v, &s.o, &s.yt, &s.hc, &s.ht, &s.oref};
    for (size_t* p : slots) {
        *p = off;
        off += round_up(s.bytes);
    }
    s.rs = off;
    off += round_up(s.rbytes);
    s.part = off;
    off += round_up(MRAE_PARTIALS * sizeof(double));
    s.res = off;
    off += ALIGN;
    s.layers = off;
    s.per_layer = round_up(s.rbytes) + round_up(s.bytes);
    s.total = off + (size_t)n_layers * s.per_layer;
    return s;
}

dfa_status err(dfa_status st, const char* what) { return (dfa_status)dfa::set_error(st, "%s", what); }

dfa_status hip(hipError_t e) {
    if (e == hipSuccess) return DFA_OK;
    return (dfa_status)dfa::set_error(DFA_ERR_HIP, "plan search: %s (%s)", hipGetErrorName(e), hipGetErrorString(e));
}

}  // namespace

extern "C" {

size_t dfa_plan_search_workspace_bytes(int n_layers, int B, int H, int L, int d) {
    if (n_layers <= 0 || B <= 0 || H <= 0 || L <= 0 || d <= 0) return 0;
    return layout(n_layers, B, H, L, d).total;
}

dfa_status dfa_mrae(const void* A, const void* B, size_t n, void* workspace, double* result, hipStream_t stream) {
    if (!A || !B || !workspace || !result) return err(DFA_ERR_INVALID_ARG, "dfa_mrae: NULL pointer");
    if ((((uintptr_t)A | (uintptr_t)B | (uintptr_t)workspace) & 15) || ((uintptr_t)result & 7))
        return err(DFA_ERR_INVALID_ARG, "dfa_mrae: A, B, workspace must be 16-byte aligned, result 8-byte aligned");
    return hip(dfa::launch_mrae(A, B, n, 1e-6f, (double*)workspace, DFA_MRAE_WORKSPACE_BYTES / sizeof(double), result,
                                stream));
}

dfa_status dfa_mrae_noalloc(const void* A, const void* B, size_t n, double* result, hipStream_t stream) {
    if (!A || !B || !result) return err(DFA_ERR_INVALID_ARG, "dfa_mrae_noalloc: NULL pointer");
    if ((((uintptr_t)A | (uintptr_t)B) & 15) || ((uintptr_t)result & 7))
        return err(DFA_ERR_INVALID_ARG, "dfa_mrae_noalloc: A and B must be 16-byte aligned, result 8-byte aligned");
    if (n > DFA_MRAE_NOALLOC_MAX_ELEMS)
        return err(DFA_ERR_INVALID_ARG, "dfa_mrae_noalloc: n exceeds DFA_MRAE_NOALLOC_MAX_ELEMS (2^40 elements)");
    // the reduction's grid is capped at the array's length: one partial sum per workgroup
    static_assert(MRAE_PARTIALS == dfa::MRAE_SCRATCH_PARTIALS, "same grid as dfa_mrae");
    if (dfa::mrae_workgroups(n, MRAE_PARTIALS) > (size_t)dfa::MRAE_SCRATCH_PARTIALS)
        return err(DFA_ERR_INVALID_ARG, "dfa_mrae_noalloc: more partial sums than the scratch array holds");
    double* part = nullptr;
    dfa_status st = hip(dfa::scratch_partials(&part));
    if (st != DFA_OK) return st;
    return hip(dfa::launch_mrae(A, B, n, 1e-6f, part, MRAE_PARTIALS, result, stream));
}

dfa_status dfa_plan_search(int n_layers, int n_steps, const void* const* X_steps, const void* const* Wqkv,
                           const void* const* bqkv, const void* const* Wo, const void* const* bo, double delta, int B,
                           int H, int L, int d, int w, void* workspace, size_t workspace_bytes, int32_t* plan,
                           double* loss, hipStream_t stream) {
    if (n_layers <= 0 || n_steps <= 0 || B <= 0 || L <= 0 || !(delta >= 0) || w < 0)
        return err(DFA_ERR_INVALID_ARG, "dfa_plan_search: bad sizes, delta or w");
    if (!X_steps || !Wqkv || !Wo || !plan || !loss || !workspace)
        return err(DFA_ERR_INVALID_ARG, "dfa_plan_search: NULL array");
    if (!dfa::proj_shape_supported(H, d)) return err(DFA_ERR_UNSUPPORTED, "dfa_plan_search: unsupported H * d");
    const Layout s = layout(n_layers, B, H, L, d);
    if (workspace_bytes < s.total) return err(DFA_ERR_INVALID_ARG, "dfa_plan_search: workspace too small");
    if ((uintptr_t)workspace & (ALIGN - 1)) return err(DFA_ERR_INVALID_ARG, "dfa_plan_search: workspace not 256-byte aligned");
    for (int t = 0; t < n_steps; ++t)
        if (!X_steps[t]) return err(DFA_ERR_INVALID_ARG, "dfa_plan_search: NULL hidden state");
    for (int i = 0; i < n_layers; ++i)
        if (!Wqkv[i] || !Wo[i]) return err(DFA_ERR_INVALID_ARG, "dfa_plan_search: NULL weight");

    char* ws = (char*)workspace;
    void *Q = ws + s.q, *K = ws + s.k, *V = ws + s.v, *O = ws + s.o, *Yt = ws + s.yt, *Hc = ws + s.hc,
         *Ht = ws + s.ht, *Oref = ws + s.oref, *Rs = ws + s.rs;
    double* part = (double*)(ws + s.part);
    double* res = (double*)(ws + s.res);
    std::vector<void*> R(n_layers), Yc(n_layers);
    for (int i = 0; i < n_layers; ++i) {
        R[i] = ws + s.layers + (size_t)i * s.per_layer;
        Yc[i] = (char*)R[i] + round_up(s.rbytes);
    }
    const size_t n_elem = s.bytes / 2;
    const long long C = (long long)H * d;

    // strategies from the largest computation reduction to the smallest;
    // ties keep the order of the paper's list
    std::vector<int> order = {DFA_AST_REUSE, DFA_WARS_ASC_REUSE, DFA_WARS_REUSE, DFA_ASC_REUSE};
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return kept_fraction(a, L, C, w) < kept_fraction(b, L, C, w); });

    std::vector<char> has_y(n_layers, 0), has_r(n_layers, 0);
    dfa_status st;
    auto module = [&](int code, int i, const void* X, void* Rr, void* Ycache) {
        return dfa_module_step(code, X, Wqkv[i], bqkv ? bqkv[i] : nullptr, Wo[i], bo ? bo[i] : nullptr, Q, K, V, O,
                               Rr, Yt, Ycache, B, H, L, d, w, stream);
    };
    // Uncompressed layers first..n-1, applied in place to the hidden state Hs.
    // An uncompressed layer runs the same kernel as an uncompressed commit
    // (the refresh, whose output rounds differently from the full-attention
    // kernel), with a scratch residual, so that identical inputs give
    // identical outputs along every path.
    auto forward_rest = [&](int first, void* Hs) -> dfa_status {
        for (int l = first; l < n_layers; ++l) {
            dfa_status e;
            if ((e = module(DFA_WARS_REFRESH, l, Hs, Rs, nullptr)) != DFA_OK) return e;
            if ((e = hip(dfa::launch_add_bf16(Hs, Yt, Hs, n_elem, stream))) != DFA_OK) return e;
        }
        return DFA_OK;
    };
    auto loss_vs_ref = [&](const void* out, double* v) -> dfa_status {
        dfa_status e;
        if ((e = hip(dfa::launch_mrae(Oref, out, n_elem, 1e-6f, part, MRAE_PARTIALS, res, stream))) != DFA_OK) return e;
        if ((e = hip(hipMemcpyAsync(v, res, sizeof(double), hipMemcpyDeviceToHost, stream))) != DFA_OK) return e;
        return hip(hipStreamSynchronize(stream));
    };
    auto applicable = [&](int code, int i) {
        if (code == DFA_AST_REUSE) return (bool)has_y[i];
        if (code == DFA_WARS_REUSE) return (bool)has_r[i];
        if (code == DFA_WARS_ASC_REUSE) return has_r[i] && B % 2 == 0;
        return B % 2 == 0;   // ASC
    };

    for (int t = 0; t < n_steps; ++t) {
        // output of the uncompressed model at this step
        if ((st = hip(hipMemcpyAsync(Oref, X_steps[t], s.bytes, hipMemcpyDeviceToDevice, stream))) != DFA_OK) return st;
        if ((st = forward_rest(0, Oref)) != DFA_OK) return st;
        if ((st = hip(hipMemcpyAsync(Hc, X_steps[t], s.bytes, hipMemcpyDeviceToDevice, stream))) != DFA_OK) return st;
        for (int i = 0; i < n_layers; ++i) {
            const double thr = (double)(i + 1) / n_layers * delta;
            int chosen = DFA_WARS_REFRESH;
            double chosen_loss = NAN;
            for (int m : order) {
                if (!applicable(m, i)) continue;
                // layer i alone compressed with m on top of the choices for
                // layers < i (already applied to Hc); the caches are only read
                if ((st = module(m, i, Hc, R[i], m == DFA_AST_REUSE ? Yc[i] : nullptr)) != DFA_OK) return st;
                if ((st = hip(dfa::launch_add_bf16(Hc, Yt, Ht, n_elem, stream))) != DFA_OK) return st;
                if ((st = forward_rest(i + 1, Ht)) != DFA_OK) return st;
                double lv;
                if ((st = loss_vs_ref(Ht, &lv)) != DFA_OK) return st;
                if (lv < thr) {
                    chosen = m;
                    chosen_loss = lv;
                    break;
                }
            }
            // commit layer i: its caches now follow the chosen strategy
            if ((st = module(chosen, i, Hc, R[i], Yc[i])) != DFA_OK) return st;
            if ((st = hip(dfa::launch_add_bf16(Hc, Yt, Hc, n_elem, stream))) != DFA_OK) return st;
            has_y[i] = 1;
            if (chosen == DFA_WARS_REFRESH) has_r[i] = 1;
            plan[(size_t)t * n_layers + i] = chosen;
            loss[(size_t)t * n_layers + i] = chosen_loss;
        }
    }
    return hip(hipStreamSynchronize(stream));
}

}  // extern "C"
