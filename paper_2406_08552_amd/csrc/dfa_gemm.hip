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
// or 256 tokens (the larger tile when the grid still has four rounds of work
// per CU) and walks K in tiles of 64 or 32.  The 128-token tile loads the
// next k-tile from global memory into registers while the MFMAs consume the
// current one from LDS, then stores it into the other LDS buffer (double
// buffering, one barrier per k-tile).  The 256-token tile streams its k-tiles
// through a ring of three LDS stages with direct global -> LDS copies issued
// two k-tiles ahead (one barrier per k-tile, a partial vmcnt wait).  Each wavefront owns 64 features x 64 or 128 tokens as blocks
// of v_mfma_f32_32x32x16_bf16 (operand layouts: lane l, h = l / 32, A element
// e = A[l % 32][8h + e], B element e = B[8h + e][l % 32], output element
// i = D[8 (i/4) + 4h + i%4][l % 32]).  The 128-token tile's LDS rows carry one
// 16-byte pad chunk (144-byte pitch); the 256-token tile's 64-byte rows are
// swizzled instead (chunk_off).  Either way the staging stores and the 16-byte
// operand reads are free of bank conflicts.  Blocks are remapped so that each XCD works
// through a contiguous range of token tiles with all their feature tiles,
// keeping the token tile's activations in that XCD's L2 (with weights larger
// than an L2, in groups of 8 token tiles: launch_gemm).
//
// Measured at 32768 tokens x 1152 features (PixArt-Sigma at 2048 px), against
// earlier forms of this kernel: scattering 8-byte pieces straight from the
// accumulators cost about a quarter of the QKV projection's time; direct
// global->LDS copies were no faster than register staging; the 256-token
// tile takes about 10% off the QKV projection; its swizzled rows, against
// 80-byte padded ones, cut LDS bank-conflict cycles from 14% to 1.4% and took
// 2% more off it.  Larger tiles still
// (192 x 256 at one wavefront per SIMD, also with a four-stage copy ring)
// did not beat these shapes.
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
constexpr int TILE_FEW = 0, TILE_MANY = 1;       // workgroup tile shapes (see Tile)

// Workgroup tile shape.  TILE_FEW: 128 tokens, k-tiles of 64 (144-byte LDS
// rows); TILE_MANY: 256 tokens, k-tiles of 32 (64-byte swizzled rows), which moves a
// quarter fewer bytes into the CUs per FLOP but needs more workgroups to fill
// the chip.  Both sum over k in the same order, so they give identical results.
template <int SHAPE>
struct Tile {
    static constexpr int BT = SHAPE == TILE_MANY ? 4 : 2;     // 32-token blocks per wavefront
    static constexpr int GTOK = 64 * BT;                       // tokens per workgroup
    static constexpr int GK = SHAPE == TILE_MANY ? 32 : 64;    // k per LDS tile
    static constexpr int GCH = GK / 8;                         // 16-byte chunks of data per row
    static constexpr bool SWZ = SHAPE == TILE_MANY;            // swizzled 64-byte rows instead of a pad chunk
    static constexpr int GP = (GCH + (SWZ ? 0 : 1)) * 8;       // row pitch in elements
    static constexpr int ATILE = GF * GP;                      // W tile
    static constexpr int STAGE = (GF + GTOK) * GP;             // W tile, then activation tile
    static constexpr int OP = GF + 8;                          // output staging row pitch (elements)
    static constexpr int ACH = GF * GCH / GT;                  // W chunks per thread and k-tile
    static constexpr int BCH = GTOK * GCH / GT;                // activation chunks per thread and k-tile
    // the 256-token tile streams its k-tiles through a ring of three LDS stages
    // filled by direct global -> LDS copies two k-tiles ahead (RING); the
    // 128-token tile stages them through registers into two LDS buffers
    static constexpr bool RING = SHAPE == TILE_MANY;
    static constexpr int NSTAGE = RING ? 3 : 2;
    static constexpr int SMEM = NSTAGE * STAGE > GTOK * OP ? NSTAGE * STAGE : GTOK * OP;
    static_assert(GF * GCH % GT == 0 && GTOK * GCH % GT == 0, "chunks per thread");
    static_assert((size_t)SMEM * sizeof(uint16_t) * 2 <= 160 * 1024, "two workgroups per CU must fit in LDS");
};

// Element offset of 16-byte chunk ch of LDS row row.  Padded rows keep the
// chunk in place.  Swizzled rows (four chunks, 64 bytes) move it to
// ch ^ s(row), s(row) = bits 2-3 of row in reverse order: the staging stores
// (whole rows) and the operand reads (one chunk of 32 consecutive rows per
// half-wavefront) then both fall on distinct bank groups, where a 16-byte pad
// on 64-byte rows leaves the stores with conflicts.
template <int SHAPE>
__device__ __forceinline__ int chunk_off(int row, int ch) {
    using T = Tile<SHAPE>;
    if constexpr (T::SWZ) return row * T::GP + ((ch ^ (((row >> 1) & 2) | ((row >> 3) & 1))) << 3);
    return row * T::GP + ch * 8;
}

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
    int group;               // token tiles per group of the block order (1: all feature tiles of a token tile in turn)
    int nblocks;
};

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, bf16x2{(__bf16)lo, (__bf16)hi});
}

// Global -> register loads of k-tile kt: thread tid owns chunks
// c = it * GT + tid of the W tile and of the activation tile, chunk c being
// row c / GCH, 16-byte column c % GCH.  Token rows beyond M load row M - 1
// (their outputs are not stored).
template <int ACT, int SHAPE>
__device__ __forceinline__ void load_gemm_tile(const GemmParams& p, int n0, int t0, int kt, int tid,
                                               u32x4 (&r)[Tile<SHAPE>::ACH + Tile<SHAPE>::BCH]) {
    using T = Tile<SHAPE>;
#pragma unroll
    for (int it = 0; it < T::ACH; ++it) {
        const int c = it * GT + tid;
        const int row = c / T::GCH, ch = c % T::GCH;
        r[it] = *(const u32x4*)(p.W + (size_t)(n0 + row) * p.K + kt * T::GK + ch * 8);
    }
#pragma unroll
    for (int it = 0; it < T::BCH; ++it) {
        const int c = it * GT + tid;
        const int row = c / T::GCH, ch = c % T::GCH;
        const int kk = kt * T::GK + ch * 8;
        const int t = min(t0 + row, p.M - 1);
        const uint16_t* src;
        if constexpr (ACT == ACT_ROWS) {
            src = p.act + (size_t)t * p.K + kk;
        } else {
            const int b = t / p.L, l = t - b * p.L;
            const int h = kk / p.d, j = kk - h * p.d;
            src = p.act + ((size_t)(b * p.H + h) * p.L + l) * p.d + j;
        }
        r[T::ACH + it] = *(const u32x4*)src;
    }
}

// Direct global -> LDS copy of k-tile kt into one stage (RING tiles): the
// stage's 16-byte slots are filled in order, lane l of a copy writing slot
// base + l, so each lane loads the chunk that the swizzle places in its slot
// (slot P holds chunk (P & 3) ^ s(row) of row P >> 2).  Token rows beyond M
// copy row M - 1 (their outputs are not stored).
template <int ACT, int SHAPE>
__device__ __forceinline__ void issue_gemm_tile(const GemmParams& p, int n0, int t0, int kt, int tid, uint16_t* As) {
    using T = Tile<SHAPE>;
    static_assert(T::SWZ && T::GCH == 4 && T::GP == 32, "ring tiles are swizzled 64-byte rows");
    const int wave_slot0 = __builtin_amdgcn_readfirstlane(tid & ~63);
#pragma unroll
    for (int it = 0; it < T::ACH + T::BCH; ++it) {
        const int slot = it * GT + tid;          // 16-byte slot of the stage (W rows first)
        const int row = slot >> 2;
        const int ch = (slot & 3) ^ (((row >> 1) & 2) | ((row >> 3) & 1));
        const int kk = kt * T::GK + ch * 8;
        const uint16_t* src;
        if (row < GF) {
            src = p.W + (size_t)(n0 + row) * p.K + kk;
        } else {
            const int t = min(t0 + row - GF, p.M - 1);
            if constexpr (ACT == ACT_ROWS) {
                src = p.act + (size_t)t * p.K + kk;
            } else {
                const int b = t / p.L, l = t - b * p.L;
                const int h = kk / p.d, j = kk - h * p.d;
                src = p.act + ((size_t)(b * p.H + h) * p.L + l) * p.d + j;
            }
        }
        __builtin_amdgcn_global_load_lds((const void*)src,
                                         (__attribute__((address_space(3))) void*)(As + 8 * (it * GT + wave_slot0)), 16, 0,
                                         0);
    }
}

template <int SHAPE>
__device__ __forceinline__ void store_gemm_tile(int tid, const u32x4 (&r)[Tile<SHAPE>::ACH + Tile<SHAPE>::BCH],
                                                uint16_t* As, uint16_t* Bs) {
    using T = Tile<SHAPE>;
#pragma unroll
    for (int it = 0; it < T::ACH; ++it) {
        const int c = it * GT + tid;
        *(u32x4*)(As + chunk_off<SHAPE>(c / T::GCH, c % T::GCH)) = r[it];
    }
#pragma unroll
    for (int it = 0; it < T::BCH; ++it) {
        const int c = it * GT + tid;
        *(u32x4*)(Bs + chunk_off<SHAPE>(c / T::GCH, c % T::GCH)) = r[T::ACH + it];
    }
}

template <int ACT, int OUT, int SHAPE>
__global__ void __launch_bounds__(GT) __attribute__((amdgpu_waves_per_eu(2, 2))) gemm_kernel(GemmParams p) {
    using T = Tile<SHAPE>;
    constexpr int BT = T::BT, GK = T::GK, GP = T::GP, GTOK = T::GTOK;
    __shared__ __attribute__((aligned(16))) uint16_t smem[T::SMEM];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wf = wave & 1, wt = wave >> 1;    // the wavefront's feature and token halves
    const int r32 = lane & 31, h = lane >> 5;

    int blk = blockIdx.x;
    if ((p.nblocks & 7) == 0) blk = (blk & 7) * (p.nblocks >> 3) + (blk >> 3);
    // groups of p.group token tiles, each group's blocks feature tile by
    // feature tile (a bijection onto the tiles; the last group may be short)
    const int ntt = p.nblocks / p.nft;
    const int grp = blk / (p.group * p.nft), rem = blk - grp * (p.group * p.nft);
    const int gc = min(p.group, ntt - grp * p.group);
    const int ft = rem / gc, tt = grp * p.group + rem % gc;
    const int n0 = ft * GF, t0 = tt * GTOK;

    f32x16 acc[2][BT];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < BT; ++nb)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[mb][nb][i] = 0.f;

    const int nk = p.K / GK;
    // one k-tile of MFMAs from LDS stage As / Bs
    auto mma_tile = [&](const uint16_t* As, const uint16_t* Bs) {
#pragma unroll
        for (int ks = 0; ks < GK / 16; ++ks) {
            const uint16_t* arow = As + chunk_off<SHAPE>(64 * wf + r32, 2 * ks + h);
            const uint16_t* brow = Bs + chunk_off<SHAPE>(32 * BT * wt + r32, 2 * ks + h);
            bf16x8 a[2], b[BT];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) a[mb] = __builtin_bit_cast(bf16x8, *(const u32x4*)(arow + 32 * mb * GP));
#pragma unroll
            for (int nb = 0; nb < BT; ++nb) b[nb] = __builtin_bit_cast(bf16x8, *(const u32x4*)(brow + 32 * nb * GP));
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < BT; ++nb)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mb], b[nb], acc[mb][nb], 0, 0, 0);
        }
    };
    if constexpr (T::RING) {
        // k-tiles kt + 1 and kt + 2 are in flight while kt is used; each
        // thread issues ACH + BCH copies per k-tile, so vmcnt(ACH + BCH)
        // leaves only the newer k-tile outstanding
        issue_gemm_tile<ACT, SHAPE>(p, n0, t0, 0, tid, smem);
        if (nk > 1) issue_gemm_tile<ACT, SHAPE>(p, n0, t0, 1, tid, smem + T::STAGE);
        for (int kt = 0; kt < nk; ++kt) {
            static_assert(T::ACH + T::BCH < 16, "vmcnt immediate");
            if (kt + 1 < nk) __builtin_amdgcn_s_waitcnt(0x0F70 | (T::ACH + T::BCH));
            else __builtin_amdgcn_s_waitcnt(0x0F70);
            // every copy of k-tile kt has landed, and every wavefront is done
            // with the stage k-tile kt + 2 overwrites (the one k-tile kt - 1 used)
            __syncthreads();
            if (kt + 2 < nk) issue_gemm_tile<ACT, SHAPE>(p, n0, t0, kt + 2, tid, smem + ((kt + 2) % 3) * T::STAGE);
            const uint16_t* As = smem + (kt % 3) * T::STAGE;
            mma_tile(As, As + T::ATILE);
        }
        __syncthreads();
    } else {
    int stage = 0;
    u32x4 stg[T::ACH + T::BCH];
    load_gemm_tile<ACT, SHAPE>(p, n0, t0, 0, tid, stg);
    store_gemm_tile<SHAPE>(tid, stg, smem, smem + T::ATILE);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const uint16_t* As = smem + stage * T::STAGE;
        const uint16_t* Bs = As + T::ATILE;
        if (kt + 1 < nk) load_gemm_tile<ACT, SHAPE>(p, n0, t0, kt + 1, tid, stg);
#pragma unroll
        for (int ks = 0; ks < GK / 16; ++ks) {
            // operand rows differ from the lane's first row by multiples of 32,
            // which leave the swizzle unchanged
            const uint16_t* arow = As + chunk_off<SHAPE>(64 * wf + r32, 2 * ks + h);
            const uint16_t* brow = Bs + chunk_off<SHAPE>(32 * BT * wt + r32, 2 * ks + h);
            bf16x8 a[2], b[BT];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) a[mb] = __builtin_bit_cast(bf16x8, *(const u32x4*)(arow + 32 * mb * GP));
#pragma unroll
            for (int nb = 0; nb < BT; ++nb) b[nb] = __builtin_bit_cast(bf16x8, *(const u32x4*)(brow + 32 * nb * GP));
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < BT; ++nb)
                    acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mb], b[nb], acc[mb][nb], 0, 0, 0);
        }
        if (kt + 1 < nk) {
            uint16_t* An = smem + (stage ^ 1) * T::STAGE;
            store_gemm_tile<SHAPE>(tid, stg, An, An + T::ATILE);
        }
        __syncthreads();
        stage ^= 1;
    }
    }

    // epilogue: bias and bf16 rounding, then the tile goes through LDS as
    // [token][feature] rows so that the stores are 16-byte chunks in row
    // order (the loop ended on a barrier, so every stage is free)
    uint16_t* ot = smem;
#pragma unroll
    for (int nb = 0; nb < BT; ++nb) {
        const int tl = 32 * BT * wt + 32 * nb + r32;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                const int fl = 64 * wf + 32 * mb + 8 * jb + 4 * h;
                f32x4 v{acc[mb][nb][4 * jb], acc[mb][nb][4 * jb + 1], acc[mb][nb][4 * jb + 2], acc[mb][nb][4 * jb + 3]};
                if (p.bias) v += *(const f32x4*)(p.bias + n0 + fl);
                *(u32x2*)(ot + tl * T::OP + fl) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
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
        const u32x4 val = *(const u32x4*)(ot + tl * T::OP + 8 * g);
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

template <int ACT, int OUT, int SHAPE>
hipError_t launch_shape(GemmParams& p, hipStream_t stream) {
    constexpr int GTOK = Tile<SHAPE>::GTOK;
    const long long nb = (long long)((p.M + GTOK - 1) / GTOK) * p.nft;
    if (nb <= 0 || nb > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    p.nblocks = (int)nb;
    hipLaunchKernelGGL((gemm_kernel<ACT, OUT, SHAPE>), dim3(p.nblocks), dim3(GT), 0, stream, p);
    return hipGetLastError();
}

// The 256-token tile when it still gives every CU at least four rounds of two
// workgroups (measured at 32768 tokens: the QKV projection gains about 10%
// with it, the output projection, 2.25 rounds, loses about as much).
// Block order: a weight that fits one XCD's 4 MB L2 stays there while an XCD
// walks all feature tiles of one token tile after another.  A larger weight
// (the QKV projection's 7.6 MB at C = 1152) would then be fetched again for
// every token tile, so the blocks go in groups of 8 token tiles, feature tile
// by feature tile: an XCD's resident workgroups then share both operands'
// tiles (measured at 32768 tokens: fetched bytes 936 -> 643 MB, time -5%; the
// output projection's 2.6 MB weight fetched more and ran 1% slower grouped).
template <int ACT, int OUT>
hipError_t launch_gemm(GemmParams& p, hipStream_t stream) {
    p.nft = p.N / GF;
    p.group = (long long)p.N * p.K * 2 > (4LL << 20) ? 8 : 1;
    const long long many = (long long)((p.M + Tile<TILE_MANY>::GTOK - 1) / Tile<TILE_MANY>::GTOK) * p.nft;
    if (many >= 4LL * 2 * 256) return launch_shape<ACT, OUT, TILE_MANY>(p, stream);
    return launch_shape<ACT, OUT, TILE_FEW>(p, stream);
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
