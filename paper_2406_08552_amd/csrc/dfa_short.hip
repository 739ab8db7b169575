// Attention kernels for short sequences (L <= 32) on gfx950 (CDNA4): the same
// three operations as the tiled kernels, for workloads made of many short
// sequences, such as temporal attention across the frames of a video DiT
// (one sequence per spatial position and head):
//   MODE_FULL     O = softmax(Q K^T / sqrt(d)) V                 (Sec. 3.2, Eq. 1 first line)
//   MODE_REFRESH  O = full attention, R = O - window attention    (Sec. 3.2, Eq. 1), R in fp32
//   MODE_WINDOW   O = window attention (+ R when given)           (Sec. 3.2, Eq. 2)
// The window is the band |i - j| <= w over the token index of the sequence.
//
// Work decomposition
//   One wavefront owns one whole (batch, head) sequence: its queries are
//   NB 16-query MFMA blocks and its keys one 16 * NB-key tile, so softmax is
//   exact (no running maximum) and each sequence is read once.  The tiled
//   kernels give a workgroup 128 queries and 64-key tiles, which leaves most
//   of each workgroup idle when L is 16.
//
// MFMA mapping (v_mfma_f32_16x16x32_bf16, fp32 accumulation), as in the
// tiled kernels: scores are formed transposed, S^T = K Q^T, with both
// operands loaded straight from global memory in the operand layout (lane l
// holds 8 consecutive dims of row l % 16); the probabilities, rounded to
// bf16, are the B operand of O^T = V^T P^T, whose A operand comes from the
// wavefront's row-major copy of V in LDS through transposing reads.  Keys of
// the 32-key PV chunk at or beyond L have zero probability and zero V rows.
// For d = 72 the LDS column 72 of V holds 1.0, so the PV product also yields
// the softmax row sum of the same bf16 probabilities that weight V.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dfa_internal.h"

namespace dfa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int SW = 4;                      // wavefronts (sequences) per workgroup
constexpr float NEG_INF = -__builtin_inff();

enum { MODE_FULL = 0, MODE_REFRESH = 1, MODE_WINDOW = 2, MODE_ASC = 3 };
// MODE_ASC computes exactly what MODE_FULL computes; it is a separate
// instantiation so that profiles report it apart from full attention.

template <int D>
struct SGeo {
    static_assert(D == 64 || D == 72, "head dim");
    static constexpr int NC32 = D / 32;             // k=32 chunks of the score product
    static constexpr int D32 = NC32 * 32;
    static constexpr int TAIL = D - D32;            // 0 or 8 dims in one zero-padded k=32 chunk
    static constexpr int NDB = (D + 15) / 16;       // 16-dim output blocks of PV
    static constexpr bool ONES = (D % 16) != 0;     // LDS column D of V carries ones
    static constexpr int NCH = D / 8;               // 16-byte chunks per row of Q, K, V
    static constexpr int VP = NDB * 16 + 8;         // LDS row pitch of V (elements)
    static constexpr int VCH = VP / 8;              // 16-byte chunks per LDS row
    static_assert(VP % 8 == 0 && VCH > NCH, "V pitch");
};

struct SParams {
    const uint16_t* Q;
    const uint16_t* K;
    const uint16_t* V;
    const float* Rin;         // MODE_WINDOW: fp32 residual added to the output (or null)
    float* Rout;              // MODE_REFRESH: fp32 residual output
    uint16_t* dst[4];         // every destination receives the same output
    int ndst;
    int nseq;                 // B * H sequences of L tokens
    int L, w;
    float c;                  // log2(e) / sqrt(d)
};

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, bf16x2{(__bf16)lo, (__bf16)hi});
}

// acc + the two bf16 values packed in w (one dot2 with (1, 1)): the row sum
// is taken over the same rounded probabilities that weight V, so each output
// row is a convex combination of V rows (exact for a one-hot row).
__device__ __forceinline__ float pair_acc(uint32_t w, float acc) {
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, acc, false);
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) { return *(const u32x4*)p; }

// The rounding residuals lo - bf16(lo) and hi - bf16(hi) of a pair packed by
// pack_bf16x2 (exact in fp32), themselves packed to bf16.
__device__ __forceinline__ uint32_t pack_residual(float lo, float hi, uint32_t packed) {
    return pack_bf16x2(lo - __builtin_bit_cast(float, packed << 16), hi - __builtin_bit_cast(float, packed & 0xFFFF0000u));
}

// Probabilities of one query block (lane: query 16 qb + r, keys 16 kb + 4 g + i)
// under the key set of BAND (all keys < L, or also |i - j| <= w), packed as
// two PV B operands: the bf16 values, and `res`, their rounding residuals in
// bf16.  A row has at most 32 keys here, too few to average the bf16
// rounding of its weights (up to 2^-8 max|v - o| per output); the two
// products together apply each weight to about 2^-16 relative.  psum gets the
// fp32 sum of both packed operands over the lane's keys.
template <int NB, bool BAND>
__device__ __forceinline__ bf16x8 probs(const f32x4 (&s)[NB], int qi, int g, int L, int w, float c, float& psum,
                                        bf16x8& res) {
    float v[NB][4];
    float mx = NEG_INF;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = 16 * kb + 4 * g + i;
            bool ok = j < L;
            if constexpr (BAND) ok = ok && (qi > j ? qi - j : j - qi) <= w;
            v[kb][i] = ok ? s[kb][i] : NEG_INF;
            mx = fmaxf(mx, v[kb][i]);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // a query row beyond L may have no key in its band; its output is never stored
    const float negm = mx == NEG_INF ? 0.f : -mx * c;
    uint32_t wd[4] = {0u, 0u, 0u, 0u}, rd[4] = {0u, 0u, 0u, 0u};
    psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) {
        float p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(v[kb][i], c, negm));
        wd[2 * kb + 0] = pack_bf16x2(p[0], p[1]);
        wd[2 * kb + 1] = pack_bf16x2(p[2], p[3]);
        rd[2 * kb + 0] = pack_residual(p[0], p[1], wd[2 * kb + 0]);
        rd[2 * kb + 1] = pack_residual(p[2], p[3], wd[2 * kb + 1]);
        psum = pair_acc(wd[2 * kb + 1], pair_acc(wd[2 * kb], psum));
        psum = pair_acc(rd[2 * kb + 1], pair_acc(rd[2 * kb], psum));
    }
    res = __builtin_bit_cast(bf16x8, u32x4{rd[0], rd[1], rd[2], rd[3]});
    return __builtin_bit_cast(bf16x8, u32x4{wd[0], wd[1], wd[2], wd[3]});
}

// Register budget: at least four wavefronts per SIMD (128 VGPRs), which these
// memory-bound kernels fit without spills, except the two-block window form,
// which spills under that cap and keeps the compiler's own choice.  Measured
// against the unconstrained build: window attention at L = 16 15% faster
// (132 -> 76 VGPRs, three -> six wavefronts per SIMD), L = 12 5-10% faster in
// every mode, the L = 32 refresh 8% faster; the L = 32 window 11% slower.
template <int NB, int KMODE>
constexpr int short_min_waves() { return NB == 2 && KMODE == MODE_WINDOW ? 1 : 4; }

template <int D, int NB, int KMODE>
__global__ void __launch_bounds__(SW * 64) __attribute__((amdgpu_waves_per_eu(short_min_waves<NB, KMODE>())))
short_attn_kernel(SParams p) {
    using G = SGeo<D>;
    constexpr int MODE = KMODE == MODE_ASC ? MODE_FULL : KMODE;
    constexpr int ROWS = 16 * NB;
    __shared__ __attribute__((aligned(16))) uint16_t smem[SW * ROWS * G::VP];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int seq = blockIdx.x * SW + wave;
    if (seq >= p.nseq) return;   // wave-uniform; the kernel has no workgroup barrier
    const int r = lane & 15, g = lane >> 4;
    const int L = p.L, w = p.w;
    const float c = p.c;
    const size_t off = (size_t)seq * L * D;
    const uint16_t* __restrict__ Qs = p.Q + off;
    const uint16_t* __restrict__ Ks = p.K + off;
    const uint16_t* __restrict__ Vs = p.V + off;
    uint16_t* Vl = smem + wave * ROWS * G::VP;

    // V rows into this wavefront's LDS rows: rows at or beyond L are zero,
    // chunk NCH is (1, 0, ..., 0) for d = 72 (row-sum column), later chunks
    // zero.  Every load is issued before the first LDS write.
    constexpr int VIT = (ROWS * G::VCH + 63) / 64;
    u32x4 vv[VIT];
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
        const int idx = it * 64 + lane;
        const int row = idx / G::VCH, ch = idx - row * G::VCH;
        vv[it] = u32x4{0u, 0u, 0u, 0u};
        if (idx < ROWS * G::VCH) {
            if (ch < G::NCH) {
                if (row < L) vv[it] = load16(Vs + (size_t)row * D + 8 * ch);
            } else if (G::ONES && ch == G::NCH) {
                vv[it] = u32x4{0x3F80u, 0u, 0u, 0u};
            }
        }
    }
    // the residual of a window step, fetched early: lane (query 16 qb + r,
    // dims 16 mb + 4 g ..)
    f32x4 rin[MODE == MODE_WINDOW ? NB : 1][G::NDB];
    if constexpr (MODE == MODE_WINDOW) {
#pragma unroll
        for (int qb = 0; qb < NB; ++qb)
#pragma unroll
            for (int mb = 0; mb < G::NDB; ++mb) {
                const int qi = 16 * qb + r, col = 16 * mb + 4 * g;
                rin[qb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (p.Rin && qi < L && col < D) rin[qb][mb] = *(const f32x4*)(p.Rin + off + (size_t)qi * D + col);
            }
    }

    // S^T = K Q^T for every (query block, key block), zero rows beyond L
    f32x4 S[NB][NB];
    {
        bf16x8 qa[NB][G::NC32], qt[NB];
#pragma unroll
        for (int qb = 0; qb < NB; ++qb) {
            const int row = 16 * qb + r;
            const bool ok = row < L;
#pragma unroll
            for (int cc = 0; cc < G::NC32; ++cc)
                qa[qb][cc] = __builtin_bit_cast(bf16x8, ok ? load16(Qs + (size_t)row * D + 32 * cc + 8 * g) : u32x4{0u, 0u, 0u, 0u});
            qt[qb] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
            if constexpr (G::TAIL > 0)
                if (ok && 8 * g < G::TAIL) qt[qb] = __builtin_bit_cast(bf16x8, load16(Qs + (size_t)row * D + G::D32 + 8 * g));
        }
#pragma unroll
        for (int kb = 0; kb < NB; ++kb) {
            const int row = 16 * kb + r;
            const bool ok = row < L;
            bf16x8 ka[G::NC32], kt = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
#pragma unroll
            for (int cc = 0; cc < G::NC32; ++cc)
                ka[cc] = __builtin_bit_cast(bf16x8, ok ? load16(Ks + (size_t)row * D + 32 * cc + 8 * g) : u32x4{0u, 0u, 0u, 0u});
            if constexpr (G::TAIL > 0)
                if (ok && 8 * g < G::TAIL) kt = __builtin_bit_cast(bf16x8, load16(Ks + (size_t)row * D + G::D32 + 8 * g));
#pragma unroll
            for (int qb = 0; qb < NB; ++qb) {
                f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int cc = 0; cc < G::NC32; ++cc) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[cc], qa[qb][cc], s, 0, 0, 0);
                if constexpr (G::TAIL > 0) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt, qt[qb], s, 0, 0, 0);
                S[qb][kb] = s;
            }
        }
    }

#pragma unroll
    for (int it = 0; it < VIT; ++it) {
        const int idx = it * 64 + lane;
        const int row = idx / G::VCH, ch = idx - row * G::VCH;
        if (idx < ROWS * G::VCH) *(u32x4*)(Vl + row * G::VP + 8 * ch) = vv[it];
    }

    // V^T fragments: within each 16-lane row g, lane 4m+q reads dims
    // 16mb+4q..+3 of key 4g+m (and of key 16+4g+m), every lane receiving its
    // own dim of keys 4g..4g+3 (and 16+4g..); the LDS rows were written by
    // this wavefront, whose LDS accesses complete in order
    __builtin_amdgcn_wave_barrier();
    bf16x8 va[G::NDB];
    {
        const int tm = r >> 2, tq = r & 3;
#pragma unroll
        for (int mb = 0; mb < G::NDB; ++mb) {
            const uint16_t* src = Vl + (4 * g + tm) * G::VP + 16 * mb + 4 * tq;
            const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(src));
            s16x4 v1 = s16x4{0, 0, 0, 0};
            if constexpr (NB == 2)
                v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(src + 16 * G::VP));
            va[mb] = __builtin_bit_cast(bf16x8, s16x8{v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]});
        }
    }

#pragma unroll
    for (int qb = 0; qb < NB; ++qb) {
        const int qi = 16 * qb + r;
        // one PV product per key set: [0] the set the output is stored from
        // (window for MODE_WINDOW, all keys otherwise), [1] the window of a refresh
        constexpr int NSET = MODE == MODE_REFRESH ? 2 : 1;
        f32x4 o[NSET][G::NDB];
        float inv[NSET];
#pragma unroll
        for (int set = 0; set < NSET; ++set) {
            float psum;
            bf16x8 pr;
            const bf16x8 pb = (MODE == MODE_WINDOW || set == 1) ? probs<NB, true>(S[qb], qi, g, L, w, c, psum, pr)
                                                                 : probs<NB, false>(S[qb], qi, g, L, w, c, psum, pr);
#pragma unroll
            for (int mb = 0; mb < G::NDB; ++mb) {
                o[set][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[mb], pb, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                o[set][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[mb], pr, o[set][mb], 0, 0, 0);
            }
            float l;
            if constexpr (G::ONES) {
                // row sum: output dim D of the query, held by lane 16 (D % 16 / 4) + r
                constexpr int pos = D % 16;
                l = __shfl(o[set][G::NDB - 1][pos % 4], 16 * (pos / 4) + r);
            } else {
                l = psum;
                l += __shfl_xor(l, 16);
                l += __shfl_xor(l, 32);
            }
            inv[set] = 1.f / l;
        }
        if (qi >= L) continue;
        const size_t row_off = off + (size_t)qi * D;
#pragma unroll
        for (int mb = 0; mb < G::NDB; ++mb) {
            // no fma contraction: R must be the difference of the two rounded results
#pragma clang fp contract(off)
            const int col = 16 * mb + 4 * g;
            if (col >= D) continue;
            const size_t at = row_off + col;
            const f32x4 ov = o[0][mb] * inv[0];
            f32x4 out = ov;
            if constexpr (MODE == MODE_REFRESH) *(f32x4*)(p.Rout + at) = ov - o[NSET - 1][mb] * inv[NSET - 1];
            if constexpr (MODE == MODE_WINDOW) {
                if (p.Rin) out = ov + rin[qb][mb];
            }
            const u32x2 st = u32x2{pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3])};
            for (int di = 0; di < p.ndst; ++di) *(u32x2*)(p.dst[di] + at) = st;
        }
    }
}

template <int D, int NB, int MODE>
hipError_t launch_short_attn(const AttnLaunch& a, hipStream_t stream) {
    SParams p{};
    p.Q = (const uint16_t*)a.Q;
    p.K = (const uint16_t*)a.K;
    p.V = (const uint16_t*)a.V;
    p.Rin = (const float*)a.Rin;
    p.Rout = (float*)a.Rout;
    p.ndst = a.ndst;
    for (int i = 0; i < 4; ++i) p.dst[i] = (uint16_t*)(i < a.ndst ? a.dst[i] : nullptr);
    const long long nseq = (long long)a.B * a.H;
    const long long nblocks = (nseq + SW - 1) / SW;
    if (nseq <= 0 || nblocks > 0x7FFFFFFFLL || a.L < 1 || a.L > 16 * NB) return hipErrorInvalidValue;
    p.nseq = (int)nseq;
    p.L = a.L;
    p.w = a.w;
    p.c = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
    hipLaunchKernelGGL((short_attn_kernel<D, NB, MODE>), dim3((unsigned)nblocks), dim3(SW * 64), 0, stream, p);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_short_mode(const AttnLaunch& a, hipStream_t stream) {
    const bool one = a.L <= 16;
    switch (a.d) {
        case 64: return one ? launch_short_attn<64, 1, MODE>(a, stream) : launch_short_attn<64, 2, MODE>(a, stream);
        case 72: return one ? launch_short_attn<72, 1, MODE>(a, stream) : launch_short_attn<72, 2, MODE>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_short_full(const AttnLaunch& a, hipStream_t s) { return launch_short_mode<MODE_FULL>(a, s); }
hipError_t launch_short_asc(const AttnLaunch& a, hipStream_t s) { return launch_short_mode<MODE_ASC>(a, s); }
hipError_t launch_short_refresh(const AttnLaunch& a, hipStream_t s) { return launch_short_mode<MODE_REFRESH>(a, s); }
hipError_t launch_short_window(const AttnLaunch& a, hipStream_t s) { return launch_short_mode<MODE_WINDOW>(a, s); }

}  // namespace dfa
