// Projections of the attention module for gfx950 (CDNA4): the fused QKV
// projection in front of the attention path and the output projection behind
// it (the module whose FLOPs Table 2 counts).
//
// Both are D = W Act^T with bf16 operands and fp32 accumulation:
//   W    [N][K]  weights, [out_features][in_features] (y = x W^T + b)
//   Act  token-major activations, K contiguous per token: X [M][K] for the
//        QKV projection, or the attention output O [B][H][L][d] read as the
//        [M][H * d] matrix of merged heads for the output projection
//   D    [N][M]  one output feature per row, one token per column
// The epilogue adds the bias, rounds to bf16 and passes the output tile
// through LDS as [token][feature] rows, so that it leaves as 16-byte chunks
// in row order: the QKV projection scatters each chunk of eight features
// straight into Q, K or V in the [B][H][L][d] layout of the attention kernels
// (feature f = which * C + head * d + dim, and d is a multiple of 8, so a
// chunk never straddles a head); the output projection stores token-major
// Y [M][N] to every destination given (the unconditional half of an ASC step
// is one of them).
//
// Work decomposition: a workgroup (4 wavefronts) owns 128 features x 128
// tokens and walks K in tiles of 64.  The next k-tile is loaded from global
// memory into registers while the MFMAs consume the current one from LDS,
// then stored into the other LDS buffer (double buffering, one barrier per
// k-tile).  Each wavefront owns 64 x 64 outputs as 2 x 2 blocks of
// v_mfma_f32_32x32x16_bf16 (operand layouts: lane l, h = l / 32, A element
// e = A[l % 32][8h + e], B element e = B[8h + e][l % 32], output element
// i = D[8 (i/4) + 4h + i%4][l % 32]).  LDS rows have a 144-byte pitch, so the
// 16-byte operand reads of 16 consecutive rows hit distinct bank groups.
// Blocks are remapped so that each XCD works through a contiguous range of
// token tiles with all their feature tiles, keeping the token tile's
// activations in that XCD's L2.
//
// Measured at 32768 tokens x 1152 features (PixArt-Sigma at 2048 px), against
// earlier forms of this kernel: scattering 8-byte pieces straight from the
// accumulators cost about a quarter of the QKV projection's time, and direct
// global->LDS copies were no faster than register staging here.  Larger
// workgroup tiles (192 x 256, one wavefront per SIMD, also with a four-stage
// copy ring) did not beat this shape.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dfa_internal.h"

namespace dfa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int GT = 256;                          // threads per workgroup
constexpr int GF = 128;                          // features per workgroup
constexpr int GTOK = 128;                        // tokens per workgroup
constexpr int GK = 64;                           // k per LDS tile
constexpr int GPC = 9;                           // row pitch in 16-byte chunks (8 data + 1 pad)
constexpr int GP = GPC * 8;                      // row pitch in elements
constexpr int G_TILE = 128 * GP;                 // one operand tile (128 rows)
constexpr int G_STAGE = 2 * G_TILE;              // A tile, then B tile
constexpr int G_OP = GF + 8;                     // output staging row pitch (elements)

enum { ACT_ROWS = 0, ACT_HEADS = 1 };   // activations: [M][K] rows, or O [B][H][L][d]
enum { OUT_QKV = 0, OUT_ROWS = 1 };     // epilogue: scatter to Q/K/V, or [M][N] rows

struct GemmParams {
    const uint16_t* W;
    const uint16_t* act;
    const float* bias;       // [N] or null
    uint16_t* dst[4];        // OUT_QKV: Q, K, V; OUT_ROWS: copies of Y
    int ndst;
    int M, N, K;             // tokens, output features, input features
    int L, H, d;             // token t = b * L + l; head geometry of Q/K/V/O
    int nft;                 // feature tiles
    int nblocks;
};

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, bf16x2{(__bf16)lo, (__bf16)hi});
}

// Global -> register loads of k-tile kt: thread tid owns chunks
// c = it * GT + tid of the W tile (it < 4) and of the activation tile
// (it >= 4), chunk c being row c / 8, 16-byte column c % 8.  Token rows
// beyond M load row M - 1 (their outputs are not stored).
template <int ACT>
__device__ __forceinline__ void load_gemm_tile(const GemmParams& p, int n0, int t0, int kt, int tid, u32x4 (&r)[8]) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int c = it * GT + tid;
        const int row = c >> 3, ch = c & 7;
        r[it] = *(const u32x4*)(p.W + (size_t)(n0 + row) * p.K + kt * GK + ch * 8);
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int c = it * GT + tid;
        const int row = c >> 3, ch = c & 7;
        const int kk = kt * GK + ch * 8;
        const int t = min(t0 + row, p.M - 1);
        const uint16_t* src;
        if constexpr (ACT == ACT_ROWS) {
            src = p.act + (size_t)t * p.K + kk;
        } else {
            const int b = t / p.L, l = t - b * p.L;
            const int h = kk / p.d, j = kk - h * p.d;
            src = p.act + ((size_t)(b * p.H + h) * p.L + l) * p.d + j;
        }
        r[4 + it] = *(const u32x4*)src;
    }
}

__device__ __forceinline__ void store_gemm_tile(int tid, const u32x4 (&r)[8], uint16_t* As, uint16_t* Bs) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int c = it * GT + tid;
        const int row = c >> 3, ch = c & 7;
        *(u32x4*)(As + row * GP + ch * 8) = r[it];
        *(u32x4*)(Bs + row * GP + ch * 8) = r[4 + it];
    }
}

template <int ACT, int OUT>
__global__ void __launch_bounds__(GT) __attribute__((amdgpu_waves_per_eu(2, 2))) gemm_kernel(GemmParams p) {
    __shared__ __attribute__((aligned(16))) uint16_t smem[2 * G_STAGE];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wf = wave & 1, wt = wave >> 1;    // the wavefront's 64-feature and 64-token halves
    const int r32 = lane & 31, h = lane >> 5;

    int blk = blockIdx.x;
    if ((p.nblocks & 7) == 0) blk = (blk & 7) * (p.nblocks >> 3) + (blk >> 3);
    const int ft = blk % p.nft, tt = blk / p.nft;
    const int n0 = ft * GF, t0 = tt * GTOK;

    f32x16 acc[2][2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[mb][nb][i] = 0.f;

    const int nk = p.K / GK;
    int stage = 0;
    u32x4 stg[8];
    load_gemm_tile<ACT>(p, n0, t0, 0, tid, stg);
    store_gemm_tile(tid, stg, smem, smem + G_TILE);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const uint16_t* As = smem + stage * G_STAGE;
        const uint16_t* Bs = As + G_TILE;
        if (kt + 1 < nk) load_gemm_tile<ACT>(p, n0, t0, kt + 1, tid, stg);
        const uint16_t* arow = As + (64 * wf + r32) * GP + 8 * h;
        const uint16_t* brow = Bs + (64 * wt + r32) * GP + 8 * h;
#pragma unroll
        for (int ks = 0; ks < GK / 16; ++ks) {
            bf16x8 a[2], b[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) a[mb] = __builtin_bit_cast(bf16x8, *(const u32x4*)(arow + 32 * mb * GP + 16 * ks));
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) b[nb] = __builtin_bit_cast(bf16x8, *(const u32x4*)(brow + 32 * nb * GP + 16 * ks));
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mb], b[nb], acc[mb][nb], 0, 0, 0);
        }
        if (kt + 1 < nk) {
            uint16_t* An = smem + (stage ^ 1) * G_STAGE;
            store_gemm_tile(tid, stg, An, An + G_TILE);
        }
        __syncthreads();
        stage ^= 1;
    }

    // epilogue: bias and bf16 rounding, then the tile goes through LDS as
    // [token][feature] rows so that the stores are 16-byte chunks in row
    // order (the loop ended on a barrier, so every stage is free)
    uint16_t* ot = smem;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const int tl = 64 * wt + 32 * nb + r32;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                const int fl = 64 * wf + 32 * mb + 8 * jb + 4 * h;
                f32x4 v{acc[mb][nb][4 * jb], acc[mb][nb][4 * jb + 1], acc[mb][nb][4 * jb + 2], acc[mb][nb][4 * jb + 3]};
                if (p.bias) v += *(const f32x4*)(p.bias + n0 + fl);
                *(u32x2*)(ot + tl * G_OP + fl) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
            }
        }
    }
    __syncthreads();
    const int C = p.N / 3;
#pragma unroll
    for (int it = 0; it < GTOK * GF / 8 / GT; ++it) {
        const int c = it * GT + tid;
        const int tl = c / (GF / 8), g = c % (GF / 8);
        const int t = t0 + tl;
        if (t >= p.M) continue;
        const u32x4 val = *(const u32x4*)(ot + tl * G_OP + 8 * g);
        const int f = n0 + 8 * g;
        if constexpr (OUT == OUT_QKV) {
            const int b = t / p.L, l = t - b * p.L;
            const int which = f / C, rem = f - which * C;
            const int head = rem / p.d, dim = rem - head * p.d;
            *(u32x4*)(p.dst[which] + ((size_t)(b * p.H + head) * p.L + l) * p.d + dim) = val;
        } else {
            for (int di = 0; di < p.ndst; ++di) *(u32x4*)(p.dst[di] + (size_t)t * p.N + f) = val;
        }
    }
}

template <int ACT, int OUT>
hipError_t launch_gemm(GemmParams& p, hipStream_t stream) {
    p.nft = p.N / GF;
    const long long ntt = (p.M + GTOK - 1) / GTOK;
    const long long nb = ntt * p.nft;
    if (nb <= 0 || nb > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    p.nblocks = (int)nb;
    static_assert((size_t)2 * G_STAGE * sizeof(uint16_t) * 2 <= 160 * 1024, "two workgroups per CU must fit in LDS");
    hipLaunchKernelGGL((gemm_kernel<ACT, OUT>), dim3(p.nblocks), dim3(GT), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

bool proj_shape_supported(int H, int d) { return H > 0 && (d == 64 || d == 72) && (H * d) % GF == 0; }

hipError_t launch_qkv_proj(const ProjLaunch& a, hipStream_t stream) {
    GemmParams p{};
    p.W = (const uint16_t*)a.W;
    p.act = (const uint16_t*)a.act;
    p.bias = (const float*)a.bias;
    for (int i = 0; i < 3; ++i) p.dst[i] = (uint16_t*)a.dst[i];
    p.ndst = 3;
    p.L = a.L;
    p.H = a.H;
    p.d = a.d;
    p.M = a.B * a.L;
    p.K = a.H * a.d;
    p.N = 3 * p.K;
    return launch_gemm<ACT_ROWS, OUT_QKV>(p, stream);
}

hipError_t launch_out_proj(const ProjLaunch& a, hipStream_t stream) {
    GemmParams p{};
    p.W = (const uint16_t*)a.W;
    p.act = (const uint16_t*)a.act;
    p.bias = (const float*)a.bias;
    p.ndst = a.ndst;
    for (int i = 0; i < 4; ++i) p.dst[i] = (uint16_t*)(i < a.ndst ? a.dst[i] : nullptr);
    p.L = a.L;
    p.H = a.H;
    p.d = a.d;
    p.M = a.B * a.L;
    p.K = a.H * a.d;
    p.N = p.K;
    return launch_gemm<ACT_HEADS, OUT_ROWS>(p, stream);
}

}  // namespace dfa
