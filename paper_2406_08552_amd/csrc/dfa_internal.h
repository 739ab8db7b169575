// Internal interface between the host library (argument checks, dispatch,
// plan generator) and the HIP kernels.  Not part of the public ABI.
#ifndef DFA_INTERNAL_H
#define DFA_INTERNAL_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

namespace dfa {

// One attention launch over B batch entries.  Every destination in dst[]
// receives the same output at the same element offset.
struct AttnLaunch {
    const void* Q;
    const void* K;
    const void* V;
    const void* Rin;   // window kernel: fp32 residual added to the output (may be null)
    void* Rout;        // refresh kernel: fp32 residual output
    void* dst[4];
    int ndst;
    int B, H, L, d, w;
};

// One projection launch of the attention module over B * L tokens.
//   QKV projection: act = X [B][L][H*d], W [3*H*d][H*d], dst[0..2] = Q, K, V
//   output projection: act = O [B][H][L][d], W [H*d][H*d], dst[0..ndst) = copies of Y [B][L][H*d]
struct ProjLaunch {
    const void* W;
    const void* act;
    const void* bias;   // fp32, may be null
    void* dst[4];
    int ndst;
    int B, H, L, d;
};

hipError_t launch_mrae(const void* a, const void* b, size_t n, float eps, double* partial, int max_partials,
                       double* out, hipStream_t stream);
// Workgroups (partial sums) of one MRAE reduction of n elements.
size_t mrae_workgroups(size_t n, int max_partials);
// Partial sums the allocation-free MRAE entry point keeps in device memory of
// its own (a file-scope array of dfa_reduce.hip, one per device).
constexpr int MRAE_SCRATCH_PARTIALS = 1024;
// Device address of that array on the current device (looked up once per device).
hipError_t scratch_partials(double** ptr);
hipError_t launch_add_bf16(const void* a, const void* b, void* out, size_t n, hipStream_t stream);

// Records the message returned by dfa_last_error() for a non-OK status.
int set_error(int status, const char* fmt, ...);

bool head_dim_supported(int d);
bool proj_shape_supported(int H, int d);
hipError_t launch_qkv_proj(const ProjLaunch& a, hipStream_t stream);
hipError_t launch_out_proj(const ProjLaunch& a, hipStream_t stream);
hipError_t launch_full(const AttnLaunch& a, hipStream_t stream);
hipError_t launch_asc(const AttnLaunch& a, hipStream_t stream);  // full attention, separate kernel name
hipError_t launch_refresh(const AttnLaunch& a, hipStream_t stream);
hipError_t launch_window(const AttnLaunch& a, hipStream_t stream);
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

// One-wavefront-per-sequence kernels for L <= SHORT_L_MAX (dfa_short.hip).
constexpr int SHORT_L_MAX = 32;
hipError_t launch_short_full(const AttnLaunch& a, hipStream_t stream);
hipError_t launch_short_asc(const AttnLaunch& a, hipStream_t stream);
hipError_t launch_short_refresh(const AttnLaunch& a, hipStream_t stream);
hipError_t launch_short_window(const AttnLaunch& a, hipStream_t stream);

// The attention operations: short sequences take the per-sequence kernels,
// longer ones the tiled kernels.
inline hipError_t attn_full(const AttnLaunch& a, hipStream_t s) {
    return a.L <= SHORT_L_MAX ? launch_short_full(a, s) : launch_full(a, s);
}
inline hipError_t attn_asc(const AttnLaunch& a, hipStream_t s) {
    return a.L <= SHORT_L_MAX ? launch_short_asc(a, s) : launch_asc(a, s);
}
inline hipError_t attn_refresh(const AttnLaunch& a, hipStream_t s) {
    return a.L <= SHORT_L_MAX ? launch_short_refresh(a, s) : launch_refresh(a, s);
}
inline hipError_t attn_window(const AttnLaunch& a, hipStream_t s) {
    return a.L <= SHORT_L_MAX ? launch_short_window(a, s) : launch_window(a, s);
}

}  // namespace dfa

#endif
