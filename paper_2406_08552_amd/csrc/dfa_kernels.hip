// Attention kernels of the DiTFastAttn hot path for gfx950 (CDNA4).
//
// One kernel template covers the three attention operations of the method:
//   MODE_FULL     O = softmax(Q K^T / sqrt(d)) V                 (Sec. 3.2, Eq. 1 first line)
//   MODE_REFRESH  O = full attention, R = O - window attention    (Sec. 3.2, Eq. 1), R in fp32
//   MODE_WINDOW   O = window attention (+ R when given)           (Sec. 3.2, Eq. 2)
//   MODE_WINDOW_FINE  the same for bands of at most 31 keys, with split probabilities
// The window is the band |i - j| <= w over the flattened token index.
//
// Work decomposition
//   A workgroup is 4 wavefronts and owns 128 consecutive queries of one
//   (batch, head); each wavefront owns 32 of them (two 16-query MFMA blocks,
//   QB = 2).  Launches whose tile walk is short (small L or a narrow band)
//   use QB = 1 instead: 64-query workgroups, four wavefronts per SIMD.
//   The workgroup walks key tiles of BK = 64 keys, staged in LDS with double
//   buffering (global loads of the next tile are in flight while the current
//   one is used).  A whole tile is copied from a uniform tile base plus
//   per-lane offsets that do not depend on the tile, so the copies take the
//   scalar-base addressing form and cost the softmax no VALU work; only the
//   ragged last tile clamps its rows.  Three workgroups share a CU (three wavefronts per SIMD), so
//   the MFMA work of one overlaps the softmax arithmetic of the others.
//
// MFMA mapping (v_mfma_f32_16x16x32_bf16, fp32 accumulation)
//   Scores are formed transposed, S^T = K Q^T: A = 16 keys x 32 dims from LDS,
//   B = 32 dims x 16 queries held in registers for the whole kernel.  The
//   result leaves every lane with a single query (lane % 16) and four keys
//   per 16-key block, so softmax statistics are per-lane values reduced over
//   the four 16-lane rows only (two permlane swaps).  The same registers,
//   rounded to bf16, are directly the B operand of the second product
//   O^T = V^T P^T, whose A operand is read from a transposed copy of the V
//   tile in LDS.  The output accumulator keeps the one-query-per-lane
//   layout, so the online-softmax rescale needs no data movement.
//   Head dim 72 = 2 x 32 + 8: the last 8 dims go through one more 16x16x32
//   MFMA with k zero-padded (on gfx950 the k=16 form costs about as much);
//   PV pads the 72 output dims to 5 blocks of 16.  The
//   padding row 72 of V^T is set to 1.0, so the PV product also yields the
//   softmax row sum (the sum of the same bf16 probabilities that weight V).
//   Head dim 64 has no padding row: the lanes sum the rounded probabilities
//   themselves, so both head dims normalise exactly the weights they apply.
//
// Online softmax
//   Per query a running max m (log2 domain) and accumulator (O, l).  The max
//   is updated lazily: the accumulator is rescaled only when a tile's max
//   exceeds m by more than 8 (so probabilities stay below 2^8 and the
//   rescale is almost never taken after the first tiles).  Once every query
//   of a wavefront has a running max, a tile's probabilities are formed
//   without its maxima, scaled by 2^-7 so that the margin is the top bit of
//   their bf16 exponents, and one OR over the packed words tests it; a tile
//   that reaches the margin is scored again and takes the exact form, which
//   forms the maxima across lanes and rescales.
//
// Narrow bands
//   A bf16 probability is off by up to 2^-8 of itself.  Over many keys these
//   errors average out; over a band of a few keys they do not, and the output
//   moves by up to 2^-8 max|v - o| on top of its own bf16 rounding.  Bands of
//   at most 31 keys per query therefore apply each probability twice: as its
//   bf16 value and as the bf16 rounding of its residual p - bf16(p), in two PV
//   products, so each weight is applied to about 2^-16 relative.  The refresh
//   does the same in its in-band phase, which forms W.
//
// Tile walk and band handling
//   The key tiles a workgroup visits are split into segments so that the hot
//   loop carries no mask: tiles where every score counts (PLAIN), the ragged
//   last tile (KEYS: j < L), and the tiles at the band edges, where each
//   wavefront classifies the tile against its own queries (inside the band,
//   outside, or straddling it with an element mask).
//   The window kernel visits only the tiles that intersect the workgroup's
//   band.  For L > 512 the refresh kernel runs ONE accumulator over two
//   phases: first the in-band scores of the band tiles (after which the
//   accumulator, normalised, is the window attention W; it is parked in the R
//   buffer), then every out-of-band score, which turns the same accumulator
//   into full attention.  R = O - W is formed in the epilogue.  Every score is
//   used exactly once, only the few band-edge tiles are visited twice, and no
//   second accumulator occupies registers.  Up to L = 512, where band-edge
//   tiles are most of the walk, the refresh instead keeps two accumulators
//   and visits every tile once (MODE_REFRESH_SPLIT).
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

constexpr int NWAVES = 4;
constexpr int NTHREADS = NWAVES * 64;
constexpr int BK = 64;                    // keys per tile
constexpr int NKB = BK / 16;              // 16-key blocks per tile
// A wavefront owns QB 16-query blocks (QB = 1 or 2), a workgroup bq<QB>() queries.
template <int QB>
constexpr int bq() { return NWAVES * QB * 16; }
constexpr float RESCALE_THRESH = 8.0f;    // lazy rescale margin (log2 units)
// Probabilities are formed as 2^(x - m - P_SHIFT): a probability at the rescale
// margin is then exactly 2, the smallest value whose bf16 form has the top
// exponent bit set, so one OR over the packed probabilities tests the margin.
// The power-of-two factor cancels in O / l.  The shifted exponent argument is
// rounded at a larger magnitude, which moves any probability of at least 2^-8
// of the running max by at most about 2^-21 of itself, far below its bf16
// rounding.
constexpr float P_SHIFT = RESCALE_THRESH - 1.0f;
constexpr uint32_t P_MARGIN_BITS = 0x40004000u;   // top exponent bit of both packed bf16 values
constexpr int FINE_MAX_HALF_WIDTH = 15;   // window half-widths applied with split probabilities
constexpr float NEG_INF = -__builtin_inff();

enum {
    MODE_FULL = 0, MODE_REFRESH = 1, MODE_WINDOW = 2, MODE_ASC = 3, MODE_REFRESH_SPLIT = 4, MODE_WINDOW_FINE = 5,
    MODE_REFRESH_FINE = 6
};
// MODE_ASC computes exactly what MODE_FULL computes (on the conditional half of
// the batch, storing every tile to both halves); it is a separate
// instantiation only so that profiles report it apart from full attention.
// MODE_REFRESH_SPLIT computes what MODE_REFRESH computes, in one pass with two
// accumulators instead of two phases with one (short sequences).
// MODE_REFRESH_FINE is the two-phase refresh for bands of at most 31 keys: its
// in-band phase (the window attention W) applies split probabilities, like
// MODE_WINDOW_FINE; the out-of-band phase, over all other keys, plain ones.
enum { MASK_NONE = 0, MASK_KEYS = 1, MASK_BAND_IN = 2, MASK_BAND_OUT = 3 };
enum { TILE_INSIDE = 0, TILE_OUTSIDE = 1, TILE_BOUNDARY = 2 };
// segment kinds of the tile walk
enum { SEG_PLAIN = 0, SEG_KEYS = 1, SEG_BAND_IN = 2, SEG_BAND_OUT = 3 };

// Geometry derived from the head dim.
//   LDS tiles are row-major, one key per row, filled by 16-byte direct
//   global->LDS copies (lane l of a copy lands at base + 16 l, so chunk c of a
//   tile sits at 16 c bytes).  K rows take KPC chunks (pitch 144 B for d = 64
//   and 72: 16-byte reads by 16 consecutive rows hit distinct 4-bank groups).
//   V rows take VPC chunks; for d = 72 the tenth chunk holds (1, 0, ..., 0),
//   a constant "dim 72 = 1" column that makes the PV product emit the row
//   sum.  Chunks at or beyond NCH are never copied into.
template <int D>
struct Geo {
    static_assert(D % 8 == 0 && D <= 72, "head dim must be a multiple of 8, at most 72");
    static_assert(D % 32 == 0 || D % 32 == 8 || D % 32 == 16, "unsupported head dim remainder");
    static constexpr int NC32 = D / 32;              // k=32 chunks of the score product
    static constexpr int D32 = NC32 * 32;
    static constexpr int TAIL = D - D32;             // dims left for one zero-padded k=32 chunk (0, 8, 16)
    static constexpr int NDB = (D + 15) / 16;        // 16-dim output blocks of PV
    static constexpr bool ONES = (D % 16) != 0;      // the padding column D of V carries ones
    static constexpr int NCH = D / 8;                // 16-byte chunks of data per row
    static constexpr int KPC = 9;                    // K row pitch in chunks (144 B)
    static constexpr int VPC = ONES ? NCH + 1 : 9;   // V row pitch in chunks (160 B for d = 72)
    static constexpr int KP = KPC * 8;               // pitches in elements
    static constexpr int VP = VPC * 8;
    static constexpr int KS_ELEMS = BK * KP;
    static constexpr int VS_ELEMS = BK * VP;
    static constexpr int STAGE_ELEMS = KS_ELEMS + VS_ELEMS;
    static constexpr int KROUNDS = (BK * KPC + NTHREADS - 1) / NTHREADS;
    static constexpr int VROUNDS = (BK * VPC + NTHREADS - 1) / NTHREADS;
    static_assert(NDB * 16 <= VP, "PV reads the padded dims of each V row");
    static_assert((KP / 2) % 32 == 4, "K pitch");
};

struct Params {
    const uint16_t* Q;
    const uint16_t* K;
    const uint16_t* V;
    const float* Rin;         // MODE_WINDOW: fp32 residual added to the output (or null)
    float* Rout;              // MODE_REFRESH: fp32 residual output (also parks W)
    uint16_t* dst[4];         // every destination receives the same output tile
    int ndst;
    int H, L, w;
    int n_qt;                 // query tiles per (batch, head)
    int nblocks;
    float c;                  // log2(e) / sqrt(d)
};

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
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

// The rounding residuals lo - bf16(lo) and hi - bf16(hi) of a pair packed by
// pack_bf16x2 (exact in fp32), themselves packed to bf16.
__device__ __forceinline__ uint32_t pack_residual(float lo, float hi, uint32_t packed) {
    return pack_bf16x2(lo - __builtin_bit_cast(float, packed << 16), hi - __builtin_bit_cast(float, packed & 0xFFFF0000u));
}

// s_waitcnt vmcnt(0): every global access of this wavefront has completed.
// The tile stores sit in branches that whole wavefronts skip; without this
// the compiler cannot prove at the loop head that the Q fragments have
// arrived and waits for the just-issued prefetch before the first MFMA.
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Reductions over the four 16-lane rows that hold the same query.
// v_permlane16_swap exchanges rows 1 and 3 of its first operand with rows 0
// and 2 of its second; v_permlane32_swap exchanges the upper half of the
// first with the lower half of the second.  Applied to two copies of x they
// leave each lane with its own and its partner row's value (rows r^1, then
// halves r^2).  Issued as inline assembly: the compiler's folding of the
// builtin's paired result has been seen to drop the second value.  The
// leading s_nop covers the VALU-write -> permlane-read hazard.
__device__ __forceinline__ void xchg16(uint32_t& a, uint32_t& b) {
    asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void xchg32(uint32_t& a, uint32_t& b) {
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}

__device__ __forceinline__ float group_max(float x) {
    uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
    xchg16(a, b);
    a = __builtin_bit_cast(uint32_t, fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b)));
    b = a;
    xchg32(a, b);
    return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}

__device__ __forceinline__ float group_sum(float x) {
    uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
    xchg16(a, b);
    a = __builtin_bit_cast(uint32_t, __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b));
    b = a;
    xchg32(a, b);
    return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

// One score tile, passed by value where a masked private copy is needed.
template <int QB>
struct Tile {
    f32x4 s[QB][NKB];
};

template <int D, int QB>
struct Acc {
    f32x4 o[QB][Geo<D>::NDB];   // O^T: lane holds dims 16*m + 4*g + i of query lane%16
    // The running max m (log2 domain) is kept in two derived forms:
    float negm[QB];             // -m - P_SHIFT, or -P_SHIFT while the query has seen no finite score
    float thr[QB];              // (m + RESCALE_THRESH) / c in raw score units (-inf: no m yet)
    float l[QB];                // lane-partial sum of the bf16 probabilities (unused when a ones row is present)
    bool fresh;                 // some query of the wavefront has no running max yet (wave-uniform)

    __device__ __forceinline__ void init() {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
            for (int mb = 0; mb < Geo<D>::NDB; ++mb) o[qb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            negm[qb] = -P_SHIFT;
            thr[qb] = NEG_INF;
            l[qb] = 0.f;
        }
        fresh = true;
    }
    // m of query block qb (-inf before its first finite score)
    __device__ __forceinline__ float running_max(int qb) const { return thr[qb] == NEG_INF ? NEG_INF : -(negm[qb] + P_SHIFT); }
};

template <int D, int QB>
struct QFrag {
    bf16x8 a[QB][Geo<D>::NC32 > 0 ? Geo<D>::NC32 : 1];
    bf16x8 t[QB];   // dims D32.. in lane rows g < TAIL/8, zero elsewhere
};

// Score tile S^T for the wavefront's 16 * QB queries against the 64 keys of one LDS
// stage: S[qb][kb][i] is the score of query (16*qb + lane%16) and key
// (16*kb + 4*(lane/16) + i) of the tile.
template <int D, int QB>
__device__ __forceinline__ void score_tile(const uint16_t* __restrict__ Ks, const QFrag<D, QB>& q, Tile<QB>& S, int r, int g) {
    using G = Geo<D>;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        const uint16_t* krow = Ks + (16 * kb + r) * G::KP;
        bf16x8 ka[G::NC32 > 0 ? G::NC32 : 1];
#pragma unroll
        for (int c = 0; c < G::NC32; ++c) ka[c] = as_bf16x8(*(const u32x4*)(krow + 32 * c + 8 * g));
        // tail dims: lane rows g >= TAIL/8 re-read the row's first tail chunk;
        // their Q tail fragment is zero, so those products vanish (the values
        // read belong to the same key row, so no other row's data enters)
        u32x4 kt = u32x4{0u, 0u, 0u, 0u};
        if constexpr (G::TAIL > 0) kt = *(const u32x4*)(krow + G::D32 + (8 * g < G::TAIL ? 8 * g : 0));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < G::NC32; ++c) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[c], q.a[qb][c], s, 0, 0, 0);
            if constexpr (G::TAIL > 0) s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kt), q.t[qb], s, 0, 0, 0);
            S.s[qb][kb] = s;
        }
    }
}

// Masks a score tile for one of the band or key masks (MASK_NONE: no-op).
template <int MASK, int QB>
__device__ __forceinline__ void mask_tile(Tile<QB>& S, int r, int g, int qrow0, int k0, int L, int w) {
    if constexpr (MASK != MASK_NONE) {
        // The lane's scores are the keys jbase + o, o = 16 kb + i.  Valid keys
        // (j < L) are the offsets o <= lim.  For the in-band mask the band
        // |qi - j| <= w, cut to [0, L - 1], is the offset range [a, b], tested
        // as one unsigned compare (o - a <= b - a); a query row beyond L whose
        // band holds no key gets an empty range.  The out-of-band mask keeps
        // the direct distance test: the range form's two extra live values per
        // query block cost the refresh kernel spills and time.
        const int jbase = k0 + 4 * g;
        const int lim = L - 1 - jbase;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            int lo = 0;
            uint32_t span = 0u;
            if constexpr (MASK == MASK_BAND_IN) {
                const int qi = qrow0 + 16 * qb + r;
                const int a = (qi > w ? qi - w : 0) - jbase;
                const uint32_t qpw = (uint32_t)qi + (uint32_t)w;    // < 2^32: qi < 2^31, w < 2^31
                const int b = (int)(qpw < (uint32_t)(L - 1) ? qpw : (uint32_t)(L - 1)) - jbase;
                lo = b < a ? (1 << 30) : a;
                span = b < a ? 0u : (uint32_t)(b - a);
            }
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int o = 16 * kb + i;
                    bool ok;
                    if constexpr (MASK == MASK_KEYS) ok = o <= lim;
                    else if constexpr (MASK == MASK_BAND_IN) ok = (uint32_t)(o - lo) <= span;
                    else {
                        const int j = jbase + o, qi = qrow0 + 16 * qb + r;
                        ok = j < L && (qi > j ? qi - j : j - qi) > w;
                    }
                    S.s[qb][kb][i] = ok ? S.s[qb][kb][i] : NEG_INF;
                }
            }
        }
    }
}

// Probabilities of one score tile against the running maxima, packed to bf16
// as the B operand of PV.  FINE adds a second operand, the rounding residual
// p - bf16(p) rounded to bf16, so that the two PV products apply each weight
// to about 2^-16 relative: rows with few keys do not average the bf16
// rounding of their weights.  psum: the lane-partial sums of what is applied
// (head dims without a ones row).
template <int D, int QB, bool FINE>
struct Probs {
    bf16x8 pb[QB][BK / 32];
    bf16x8 pl[FINE ? QB : 1][BK / 32];
    float psum[QB];
};

template <int D, int QB, bool FINE>
__device__ __forceinline__ void form_probs(const Acc<D, QB>& acc, const Tile<QB>& S, float c, Probs<D, QB, FINE>& P) {
    using G = Geo<D>;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const float negm = acc.negm[qb];
        float psum = 0.f;
#pragma unroll
        for (int h = 0; h < BK / 32; ++h) {
            uint32_t wds[4], rws[4];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const f32x4 s = S.s[qb][2 * h + half];
                const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[0], c, negm));
                const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[1], c, negm));
                const float p2 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2], c, negm));
                const float p3 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[3], c, negm));
                wds[2 * half + 0] = pack_bf16x2(p0, p1);
                wds[2 * half + 1] = pack_bf16x2(p2, p3);
                if constexpr (FINE) {
                    rws[2 * half + 0] = pack_residual(p0, p1, wds[2 * half + 0]);
                    rws[2 * half + 1] = pack_residual(p2, p3, wds[2 * half + 1]);
                }
                if constexpr (!G::ONES) {
                    psum = pair_acc(wds[2 * half + 1], pair_acc(wds[2 * half], psum));
                    if constexpr (FINE) psum = pair_acc(rws[2 * half + 1], pair_acc(rws[2 * half], psum));
                }
            }
            P.pb[qb][h] = as_bf16x8(u32x4{wds[0], wds[1], wds[2], wds[3]});
            if constexpr (FINE) P.pl[qb][h] = as_bf16x8(u32x4{rws[0], rws[1], rws[2], rws[3]});
        }
        P.psum[qb] = psum;
    }
}

// O^T += V^T P^T.  The A operand (16 dims x 32 keys) comes from the
// row-major V tile through transposing reads: within each 16-lane row,
// lane 4m+q addresses dims 16mb+4q..+3 of key k+m, and every lane receives
// its own dim of keys k..k+3.
template <int D, int QB, bool FINE>
__device__ __forceinline__ void apply_probs(Acc<D, QB>& acc, const Probs<D, QB, FINE>& P, const uint16_t* Vs, int r,
                                            int g) {
    using G = Geo<D>;
    if constexpr (!G::ONES) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) acc.l[qb] += P.psum[qb];
    }
    const int tm = r >> 2, tq = r & 3;
#pragma unroll
    for (int h = 0; h < BK / 32; ++h) {
#pragma unroll
        for (int mb = 0; mb < G::NDB; ++mb) {
            const uint16_t* src = Vs + (32 * h + 4 * g + tm) * G::VP + 16 * mb + 4 * tq;
            const s16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(src));
            const s16x4 v1 =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(src + 16 * G::VP));
            const bf16x8 va = __builtin_bit_cast(bf16x8, s16x8{v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]});
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                acc.o[qb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, P.pb[qb][h], acc.o[qb][mb], 0, 0, 0);
                if constexpr (FINE)
                    acc.o[qb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, P.pl[qb][h], acc.o[qb][mb], 0, 0, 0);
            }
        }
    }
}

// Online-softmax probabilities of one score tile, with the lazy rescale of the
// accumulator.  S is taken by value: the mask is applied to a private copy.
template <int D, int MASK, int QB, bool FINE>
__device__ __forceinline__ void exact_probs(Acc<D, QB>& acc, Tile<QB> S, int r, int g, int qrow0, int k0, int L, int w,
                                            float c, Probs<D, QB, FINE>& P) {
    using G = Geo<D>;
    mask_tile<MASK>(S, r, g, qrow0, k0, L, w);
    // Lazy rescale.  Each lane compares the largest of its own scores with
    // its query's threshold (m + RESCALE_THRESH) / c; only when some lane of
    // the wavefront exceeds it (one wave-uniform branch) are the exact tile
    // maxima formed over the four lanes that share a query, and the queries
    // whose maximum grew by more than the margin are rescaled.  Otherwise
    // every probability is below 2^8 (2 after the shift).
    float v[QB];
    bool hot = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        v[qb] = NEG_INF;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) v[qb] = fmaxf(v[qb], S.s[qb][kb][i]);
        hot = hot || v[qb] > acc.thr[qb];
    }
    if (__any(hot)) {
        bool unset = false;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            const float mx = group_max(v[qb]) * c;
            const float m = acc.running_max(qb);
            if (mx > m + RESCALE_THRESH) {
                const float alpha = __builtin_amdgcn_exp2f(m - mx);
#pragma unroll
                for (int mb = 0; mb < G::NDB; ++mb) acc.o[qb][mb] *= alpha;
                acc.l[qb] *= alpha;
                acc.negm[qb] = -mx - P_SHIFT;
                acc.thr[qb] = (mx + RESCALE_THRESH) / c;
            }
            unset = unset || acc.thr[qb] == NEG_INF;
        }
        acc.fresh = __any(unset);
    }
    form_probs(acc, S, c, P);
}

// The probabilities without the maxima, for a wavefront whose queries all have
// a running max: they are formed first, and one OR over their packed bf16
// words tests whether any reached the rescale margin.  Returns false if one
// did (rare after the first tiles); the caller then scores the tile again and
// takes exact_probs(), which rescales.
template <int D, int MASK, int QB, bool FINE>
__device__ __forceinline__ bool fast_probs(const Acc<D, QB>& acc, Tile<QB> S, int r, int g, int qrow0, int k0, int L,
                                           int w, float c, Probs<D, QB, FINE>& P) {
    mask_tile<MASK>(S, r, g, qrow0, k0, L, w);
    form_probs(acc, S, c, P);
    uint32_t bits = 0u;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int h = 0; h < BK / 32; ++h) {
            const u32x4 wv = __builtin_bit_cast(u32x4, P.pb[qb][h]);
            bits |= wv[0] | wv[1] | wv[2] | wv[3];
        }
    return !__any((bits & P_MARGIN_BITS) != 0u);
}

// Online-softmax update of the accumulator with one score tile, then PV.
template <int D, int MASK, int QB, bool FINE = false>
__device__ __forceinline__ void accumulate(Acc<D, QB>& acc, const Tile<QB>& S, const uint16_t* Vs, int r, int g,
                                           int qrow0, int k0, int L, int w, float c) {
    Probs<D, QB, FINE> P;
    exact_probs<D, MASK>(acc, S, r, g, qrow0, k0, L, w, c, P);
    apply_probs(acc, P, Vs, r, g);
}

// Row sum of one query block, broadcast to every lane of that query.
template <int D, int QB>
__device__ __forceinline__ float row_sum(const Acc<D, QB>& acc, int qb, int r) {
    using G = Geo<D>;
    if constexpr (G::ONES) {
        constexpr int MB = D / 16, GS = (D % 16) / 4, IS = (D % 16) % 4;
        return __shfl(acc.o[qb][MB][IS], r + 16 * GS);
    } else {
        return group_sum(acc.l[qb]);
    }
}

// Direct global -> LDS copy of one K/V tile (no staging registers).  Rows
// beyond L copy row L-1 instead: their scores are masked and their
// probabilities are zero, so any finite value will do.
template <int D>
__device__ __forceinline__ void issue_tile(const uint16_t* __restrict__ Kbh, const uint16_t* __restrict__ Vbh, int k0,
                                           int L, int tid, uint16_t* Ks, uint16_t* Vs) {
    using G = Geo<D>;
    // first chunk of this wavefront in a round: uniform, kept in a scalar
    // register so the LDS destination (M0) needs no per-copy lane read
    const int wave_chunk0 = __builtin_amdgcn_readfirstlane(tid & ~63);
    if (k0 + BK <= L) {
        // whole tile: a uniform tile base plus a per-lane offset that does not
        // depend on the tile (loop-invariant, so no address arithmetic per copy)
        const uint16_t* kb = Kbh + (size_t)k0 * D;
        const uint16_t* vb = Vbh + (size_t)k0 * D;
#pragma unroll
        for (int it = 0; it < G::KROUNDS; ++it) {
            const int c = it * NTHREADS + tid;
            const int row = c / G::KPC, ch = c % G::KPC;
            if (row < BK && ch < G::NCH)
                __builtin_amdgcn_global_load_lds((const void*)(kb + (uint32_t)(row * D + ch * 8)),
                                                 (__attribute__((address_space(3))) void*)(Ks + (it * NTHREADS + wave_chunk0) * 8),
                                                 16, 0, 0);
        }
#pragma unroll
        for (int it = 0; it < G::VROUNDS; ++it) {
            const int c = it * NTHREADS + tid;
            const int row = c / G::VPC, ch = c % G::VPC;
            if (row < BK && ch < G::NCH)
                __builtin_amdgcn_global_load_lds((const void*)(vb + (uint32_t)(row * D + ch * 8)),
                                                 (__attribute__((address_space(3))) void*)(Vs + (it * NTHREADS + wave_chunk0) * 8),
                                                 16, 0, 0);
        }
        return;
    }
#pragma unroll
    for (int it = 0; it < G::KROUNDS; ++it) {
        const int c = it * NTHREADS + tid;
        const int row = c / G::KPC, ch = c % G::KPC;
        if (row < BK && ch < G::NCH) {
            const int krow = min(k0 + row, L - 1);
            __builtin_amdgcn_global_load_lds((const void*)(Kbh + (size_t)krow * D + ch * 8),
                                             (__attribute__((address_space(3))) void*)(Ks + (it * NTHREADS + wave_chunk0) * 8),
                                             16, 0, 0);
        }
    }
#pragma unroll
    for (int it = 0; it < G::VROUNDS; ++it) {
        const int c = it * NTHREADS + tid;
        const int row = c / G::VPC, ch = c % G::VPC;
        if (row < BK && ch < G::NCH) {
            const int vrow = min(k0 + row, L - 1);
            __builtin_amdgcn_global_load_lds((const void*)(Vbh + (size_t)vrow * D + ch * 8),
                                             (__attribute__((address_space(3))) void*)(Vs + (it * NTHREADS + wave_chunk0) * 8),
                                             16, 0, 0);
        }
    }
}

// Direct global -> LDS copy of n16 16-byte chunks starting at src (the
// residual rows of a workgroup, at most NR chunks), chunk c landing at byte
// 16 c of dst.  Addressed as a uniform base plus a 32-bit lane offset formed
// here, so that no address stays live across the tile loop.
template <int NR>
__device__ __forceinline__ void issue_rows(const float* __restrict__ src, int n16, int tid, uint16_t* dst) {
    const int wave_chunk0 = __builtin_amdgcn_readfirstlane(tid & ~63);
    uint32_t off = (uint32_t)tid * 16u;
    asm volatile("" : "+v"(off));
#pragma unroll
    for (int it = 0; it < (NR + NTHREADS - 1) / NTHREADS; ++it) {
        if (it * NTHREADS + tid < n16)
            __builtin_amdgcn_global_load_lds((const void*)((const char*)src + off + (uint32_t)(it * NTHREADS * 16)),
                                             (__attribute__((address_space(3))) void*)(dst + 8 * (it * NTHREADS + wave_chunk0)),
                                             16, 0, 0);
    }
}

// Per-workgroup state of the tile walk.  FAST: the tiles of PLAIN segments
// take the fast form of the softmax update (a band segment's unmasked tiles
// keep the exact form: both forms beside the masks exceed the register budget).
template <int D, int QB, bool FAST = false>
struct Walk {
    using G = Geo<D>;
    const uint16_t* Kbh;
    const uint16_t* Vbh;
    uint16_t* smem;
    int tid, r, g, L, w, qw0, qhi_w;
    bool wave_active;
    float c;
    int stage;
    // Residual rows copied into the free LDS stage while the last tile is
    // used, so that the epilogue does not wait on their global read (null:
    // none); rpre_n16 16-byte chunks.
    const float* rpre;
    int rpre_n16;

    // Visit tiles [t0, t1) with one segment kind; `next_after` is the first
    // tile of the next non-empty segment (-1: none), prefetched while the
    // last tile of this segment is used.
    template <int KIND, bool FINE = false>
    __device__ __forceinline__ void run(Acc<D, QB>& acc, const QFrag<D, QB>& q, int t0, int t1, int next_after) {
        // the walk's last tile is peeled when residual rows are to be copied
        const int tl = (next_after < 0 && rpre) ? t1 - 1 : t1;
        for (int t = t0; t < tl; ++t) {
            const uint16_t* Ks = smem + stage * G::STAGE_ELEMS;
            const uint16_t* Vs = Ks + G::KS_ELEMS;
            const int next = (t + 1 < t1) ? t + 1 : next_after;
            if (next >= 0) {
                uint16_t* Kn = smem + (stage ^ 1) * G::STAGE_ELEMS;
                issue_tile<D>(Kbh, Vbh, next * BK, L, tid, Kn, Kn + G::KS_ELEMS);
            }
            if (wave_active) tile<KIND, FINE>(acc, q, Ks, Vs, t * BK);
            wait_vm_all();
            __syncthreads();
            stage ^= 1;
        }
        if (tl < t1 && t0 < t1) {
            const uint16_t* Ks = smem + stage * G::STAGE_ELEMS;
            const uint16_t* Vs = Ks + G::KS_ELEMS;
            issue_rows<bq<QB>() * D / 4>(rpre, rpre_n16, tid, smem + (stage ^ 1) * G::STAGE_ELEMS);
            if (wave_active) tile<KIND, FINE>(acc, q, Ks, Vs, tl * BK);
            wait_vm_all();
            __syncthreads();
            stage ^= 1;
        }
    }

    // Single pass over tiles [t0, t1) with two accumulators: the in-band
    // scores of each tile go to aw, the out-of-band ones to ax.  A tile that
    // is inside or outside the band for all of the wavefront's queries feeds
    // one of them; a band-edge tile is scored once and feeds both.
    __device__ __forceinline__ void run_split(Acc<D, QB>& aw, Acc<D, QB>& ax, const QFrag<D, QB>& q, int t0, int t1) {
        for (int t = t0; t < t1; ++t) {
            const uint16_t* Ks = smem + stage * G::STAGE_ELEMS;
            const uint16_t* Vs = Ks + G::KS_ELEMS;
            if (t + 1 < t1) {
                uint16_t* Kn = smem + (stage ^ 1) * G::STAGE_ELEMS;
                issue_tile<D>(Kbh, Vbh, (t + 1) * BK, L, tid, Kn, Kn + G::KS_ELEMS);
            }
            if (wave_active) tile_split(aw, ax, q, Ks, Vs, t * BK);
            wait_vm_all();
            __syncthreads();
            stage ^= 1;
        }
    }

    __device__ __forceinline__ int classify(int k0) const {
        const int khi = min(k0 + BK - 1, L - 1);
        const int mind = khi < qw0 ? qw0 - khi : (k0 > qhi_w ? k0 - qhi_w : 0);
        const int maxd = max(qhi_w - k0, khi - qw0);
        return maxd <= w ? TILE_INSIDE : (mind > w ? TILE_OUTSIDE : TILE_BOUNDARY);
    }

    __device__ __forceinline__ void tile_split(Acc<D, QB>& aw, Acc<D, QB>& ax, const QFrag<D, QB>& q,
                                               const uint16_t* Ks, const uint16_t* Vs, int k0) {
        const bool ragged = k0 + BK > L;
        const int cls = classify(k0);
        Tile<QB> S;
        score_tile<D>(Ks, q, S, r, g);
        if (cls == TILE_BOUNDARY) {
            accumulate<D, MASK_BAND_IN>(aw, S, Vs, r, g, qw0, k0, L, w, c);
            accumulate<D, MASK_BAND_OUT>(ax, S, Vs, r, g, qw0, k0, L, w, c);
        } else if (cls == TILE_INSIDE) {
            if (ragged) accumulate<D, MASK_KEYS>(aw, S, Vs, r, g, qw0, k0, L, w, c);
            else accumulate<D, MASK_NONE>(aw, S, Vs, r, g, qw0, k0, L, w, c);
        } else {
            if (ragged) accumulate<D, MASK_KEYS>(ax, S, Vs, r, g, qw0, k0, L, w, c);
            else accumulate<D, MASK_NONE>(ax, S, Vs, r, g, qw0, k0, L, w, c);
        }
    }

    // One update with the score tile S of the tile at k0.  With F, an unmasked
    // tile takes the fast form once every query of the wavefront has a running
    // max, and the exact form before that and when the fast form finds a
    // probability at the rescale margin (the tile is then scored again, so
    // that no second score tile stays live across the fast form).
    template <int MASK, bool FINE, bool F = FAST>
    __device__ __forceinline__ void update(Acc<D, QB>& acc, const QFrag<D, QB>& q, Tile<QB>& S, const uint16_t* Ks,
                                           const uint16_t* Vs, int k0) {
        Probs<D, QB, FINE> P;
        if constexpr (F && MASK == MASK_NONE) {
            if (acc.fresh || !fast_probs<D, MASK>(acc, S, r, g, qw0, k0, L, w, c, P)) {
                if (!acc.fresh) {
                    // a compiler barrier: the tile is read and scored again, not kept
                    asm volatile("" ::: "memory");
                    score_tile<D>(Ks, q, S, r, g);
                }
                exact_probs<D, MASK>(acc, S, r, g, qw0, k0, L, w, c, P);
            }
        } else {
            exact_probs<D, MASK>(acc, S, r, g, qw0, k0, L, w, c, P);
        }
        apply_probs(acc, P, Vs, r, g);
    }

    template <int KIND, bool FINE>
    __device__ __forceinline__ void tile(Acc<D, QB>& acc, const QFrag<D, QB>& q, const uint16_t* Ks, const uint16_t* Vs,
                                         int k0) {
        if constexpr (KIND == SEG_PLAIN) {
            Tile<QB> S;
            score_tile<D>(Ks, q, S, r, g);
            update<MASK_NONE, FINE>(acc, q, S, Ks, Vs, k0);
        } else if constexpr (KIND == SEG_KEYS) {
            Tile<QB> S;
            score_tile<D>(Ks, q, S, r, g);
            update<MASK_KEYS, FINE>(acc, q, S, Ks, Vs, k0);
        } else {
            // classify the tile against this wavefront's queries
            const bool ragged = k0 + BK > L;
            const int cls = classify(k0);
            constexpr int SKIP = (KIND == SEG_BAND_IN) ? TILE_OUTSIDE : TILE_INSIDE;
            if (cls == SKIP) return;
            Tile<QB> S;
            score_tile<D>(Ks, q, S, r, g);
            if (cls == TILE_BOUNDARY)
                update<KIND == SEG_BAND_IN ? MASK_BAND_IN : MASK_BAND_OUT, FINE>(acc, q, S, Ks, Vs, k0);
            else if (ragged)
                update<MASK_KEYS, FINE>(acc, q, S, Ks, Vs, k0);
            else
                update<MASK_NONE, FINE, false>(acc, q, S, Ks, Vs, k0);
        }
    }
};

template <int KMODE>
constexpr bool split_refresh() { return KMODE == MODE_REFRESH_SPLIT; }

// Refresh in one pass (Sec. 3.2, Eq. 1), for short sequences: W = aw / lw from the in-band scores
// alone; O combines both accumulators, each scaled from its own running max
// to the larger one.  A query whose band covers every key has no
// out-of-band score, and its O is then formed exactly as W, so R == 0.
template <int D, int QB>
__device__ __forceinline__ void refresh_split(const Params& p, uint16_t* smem, Walk<D, QB, false>& wk, const QFrag<D, QB>& q,
                                              size_t head_off, int ntiles) {
    using G = Geo<D>;
    Acc<D, QB> aw, ax;
    aw.init();
    ax.init();
    issue_tile<D>(wk.Kbh, wk.Vbh, 0, wk.L, wk.tid, smem, smem + G::KS_ELEMS);
    wait_vm_all();
    __syncthreads();
    wk.run_split(aw, ax, q, 0, ntiles);
    if (!wk.wave_active) return;
    const int r = wk.r, g = wk.g;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int qrow = wk.qw0 + 16 * qb + r;
        // row sums first: they exchange values across lanes
        const float lw = row_sum<D>(aw, qb, r), lx = row_sum<D>(ax, qb, r);
        const bool has_x = ax.thr[qb] != NEG_INF;
        const float mw = aw.running_max(qb);
        const float mx = ax.running_max(qb);
        const float mm = fmaxf(mw, mx);
        const float sw = has_x ? __builtin_amdgcn_exp2f(mw - mm) : 1.f;
        const float sx = has_x ? __builtin_amdgcn_exp2f(mx - mm) : 0.f;
        const float invw = 1.f / lw;
        const float inv = 1.f / (lw * sw + lx * sx);
        if (qrow >= wk.L) continue;
        const size_t row_off = head_off + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < G::NDB; ++mb) {
#pragma clang fp contract(off)
            const int col = 16 * mb + 4 * g;
            if (col >= D) continue;
            const size_t off = row_off + col;
            const f32x4 wv = aw.o[qb][mb] * invw;
            const f32x4 o = has_x ? (aw.o[qb][mb] * sw + ax.o[qb][mb] * sx) * inv : wv;
            *(f32x4*)(p.Rout + off) = o - wv;
            const u32x2 ov = u32x2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
            for (int di = 0; di < p.ndst; ++di) *(u32x2*)(p.dst[di] + off) = ov;
        }
    }
}

template <int D, int KMODE, int QB>
__device__ __forceinline__ void attn_body(const Params& p, uint16_t* smem) {
    using G = Geo<D>;
    constexpr int MODE = KMODE == MODE_ASC             ? MODE_FULL
                         : KMODE == MODE_REFRESH_SPLIT ? MODE_REFRESH
                         : KMODE == MODE_REFRESH_FINE  ? MODE_REFRESH
                         : KMODE == MODE_WINDOW_FINE   ? MODE_WINDOW
                                                       : KMODE;
    // split probabilities in the in-band segments (the window attention)
    constexpr bool FINE = KMODE == MODE_WINDOW_FINE || KMODE == MODE_REFRESH_FINE;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int r = lane & 15;
    const int g = lane >> 4;

    // XCD-aware block order: workgroups are dealt to the 8 XCDs round-robin,
    // so give each XCD a contiguous range of (head, query-tile) work and the
    // workgroups sharing an XCD's L2 read the same K/V.
    int blk = blockIdx.x;
    if ((p.nblocks & 7) == 0) blk = (blk & 7) * (p.nblocks >> 3) + (blk >> 3);
    const int bh = blk / p.n_qt;
    const int qt = blk % p.n_qt;
    const int L = p.L, w = p.w;
    const size_t head_off = (size_t)bh * L * D;
    const uint16_t* __restrict__ Qbh = p.Q + head_off;

    const int q0 = qt * bq<QB>();                 // workgroup's first query
    const int qw0 = q0 + wave * (QB * 16);       // wavefront's first query
    const int qhi_wg = min(q0 + bq<QB>() - 1, L - 1);
    const int qhi_w = min(qw0 + QB * 16 - 1, L - 1);

    // constant V padding chunk of every row in both stages: (1, 0, ..., 0) for
    // the row-sum column, never overwritten by the tile copies
    if constexpr (G::ONES) {
        for (int idx = tid; idx < 2 * BK * 8; idx += NTHREADS) {
            const int st = idx / (BK * 8), row = (idx / 8) % BK, e = idx % 8;
            smem[st * G::STAGE_ELEMS + G::KS_ELEMS + row * G::VP + D + e] = (e == 0) ? (uint16_t)0x3F80u : (uint16_t)0u;
        }
    }

    // Q fragments (B operand of S^T = K Q^T), zero beyond L and beyond d
    QFrag<D, QB> q;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int qrow = qw0 + 16 * qb + r;
        const bool ok = qrow < L;
        const uint16_t* qp = Qbh + (size_t)(ok ? qrow : 0) * D;
#pragma unroll
        for (int c = 0; c < G::NC32; ++c)
            q.a[qb][c] = as_bf16x8(ok ? *(const u32x4*)(qp + 32 * c + 8 * g) : u32x4{0u, 0u, 0u, 0u});
        q.t[qb] = as_bf16x8(u32x4{0u, 0u, 0u, 0u});
        if constexpr (G::TAIL > 0) {
            if (ok && 8 * g < G::TAIL) q.t[qb] = as_bf16x8(*(const u32x4*)(qp + G::D32 + 8 * g));
        }
    }

    // the fast update measured 1-2% faster in the long walks of two query
    // blocks per wavefront and about 1% slower in the short walks of one
    Walk<D, QB, QB == 2 && !split_refresh<KMODE>()> wk;
    wk.Kbh = p.K + head_off;
    wk.Vbh = p.V + head_off;
    wk.smem = smem;
    wk.tid = tid;
    wk.r = r;
    wk.g = g;
    wk.L = L;
    wk.w = w;
    wk.qw0 = qw0;
    wk.qhi_w = qhi_w;
    wk.wave_active = qw0 < L;
    wk.c = p.c;
    wk.stage = 0;
    wk.rpre = nullptr;
    wk.rpre_n16 = 0;
    // 64-query window walks take their residual rows through the LDS stage
    // that the last tile leaves free (one stage holds 64 fp32 rows of d <= 72)
    if constexpr (MODE == MODE_WINDOW && QB == 1) {
        static_assert(bq<1>() * D * 4 <= G::STAGE_ELEMS * 2, "residual rows must fit one LDS stage");
        if (p.Rin) {
            wk.rpre = p.Rin + head_off + (size_t)q0 * D;
            wk.rpre_n16 = (min(L, q0 + bq<1>()) - q0) * D / 4;
        }
    }

    // segments of the tile walk
    const int ntiles = (L + BK - 1) / BK, nfull = L / BK;
    int tb0 = 0, tb1 = ntiles - 1, m0 = 0, m1 = 0;
    if constexpr (MODE != MODE_FULL) {
        const long long klo = max(0LL, (long long)q0 - w);
        const long long khi = min((long long)L - 1, (long long)qhi_wg + w);
        tb0 = (int)(klo / BK);
        tb1 = (int)(khi / BK);
        // tiles inside the band for every query of the workgroup and not ragged
        const long long lo_key = (long long)qhi_wg - w;                      // first key every query reaches
        const long long hi_key = min((long long)q0 + w, (long long)L - 1);  // last key every query reaches
        const long long ai0 = lo_key <= 0 ? 0 : (lo_key + BK - 1) / BK;
        const long long ai1 = hi_key - (BK - 1) < 0 ? -1 : (hi_key - (BK - 1)) / BK;
        m0 = (int)min(max(ai0, (long long)tb0), (long long)tb1 + 1);
        m1 = (int)min(max(ai1 + 1, (long long)m0), (long long)tb1 + 1);
    }
    constexpr int NSEG = MODE == MODE_FULL ? 2 : (MODE == MODE_WINDOW ? 3 : 8);
    int s0[NSEG], s1[NSEG];
    if constexpr (MODE == MODE_FULL) {
        s0[0] = 0; s1[0] = nfull;              // PLAIN
        s0[1] = nfull; s1[1] = ntiles;         // KEYS
    } else {
        s0[0] = tb0; s1[0] = m0;               // BAND_IN
        s0[1] = m0; s1[1] = m1;                // PLAIN
        s0[2] = m1; s1[2] = tb1 + 1;           // BAND_IN
        if constexpr (MODE == MODE_REFRESH) {
            const int after = max(tb1 + 1, nfull);
            s0[3] = 0; s1[3] = tb0;            // PLAIN (left of the band)
            s0[4] = tb0; s1[4] = m0;           // BAND_OUT
            s0[5] = m1; s1[5] = tb1 + 1;       // BAND_OUT
            s0[6] = tb1 + 1; s1[6] = after;    // PLAIN (right of the band)
            s0[7] = after; s1[7] = ntiles;     // KEYS (ragged tile right of the band)
        }
    }
    // first tile of the first non-empty segment at or after each position
    int nxt[NSEG + 1];
    nxt[NSEG] = -1;
#pragma unroll
    for (int i = NSEG - 1; i >= 0; --i) nxt[i] = s0[i] < s1[i] ? s0[i] : nxt[i + 1];

    if constexpr (split_refresh<KMODE>()) {
        refresh_split<D, QB>(p, smem, wk, q, head_off, ntiles);
        return;
    }

    Acc<D, QB> acc;
    acc.init();

    // every workgroup has at least one key tile: the window of any query
    // contains the query itself
    issue_tile<D>(wk.Kbh, wk.Vbh, nxt[0] * BK, L, tid, smem, smem + G::KS_ELEMS);
    wait_vm_all();
    __syncthreads();

    if constexpr (MODE == MODE_FULL) {
        wk.template run<SEG_PLAIN>(acc, q, s0[0], s1[0], nxt[1]);
        wk.template run<SEG_KEYS>(acc, q, s0[1], s1[1], nxt[2]);
    } else {
        wk.template run<SEG_BAND_IN, FINE>(acc, q, s0[0], s1[0], nxt[1]);
        wk.template run<SEG_PLAIN, FINE>(acc, q, s0[1], s1[1], nxt[2]);
        wk.template run<SEG_BAND_IN, FINE>(acc, q, s0[2], s1[2], nxt[3]);
    }

    if constexpr (MODE == MODE_REFRESH) {
        // the accumulator now holds the window attention of the wavefront's
        // queries: park W (fp32) in the R buffer
        if (wk.wave_active) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) {
                const int qrow = qw0 + 16 * qb + r;
                const float inv = 1.f / row_sum<D>(acc, qb, r);
                if (qrow < L) {
#pragma unroll
                    for (int mb = 0; mb < G::NDB; ++mb) {
                        const int col = 16 * mb + 4 * g;
                        if (col < D) *(f32x4*)(p.Rout + head_off + (size_t)qrow * D + col) = acc.o[qb][mb] * inv;
                    }
                }
            }
        }
        wk.template run<SEG_PLAIN>(acc, q, s0[3], s1[3], nxt[4]);
        wk.template run<SEG_BAND_OUT>(acc, q, s0[4], s1[4], nxt[5]);
        wk.template run<SEG_BAND_OUT>(acc, q, s0[5], s1[5], nxt[6]);
        wk.template run<SEG_PLAIN>(acc, q, s0[6], s1[6], nxt[7]);
        wk.template run<SEG_KEYS>(acc, q, s0[7], s1[7], nxt[8]);
    }

    if (!wk.wave_active) return;

    // epilogue: normalise, form R, store bf16 to every destination
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int qrow = qw0 + 16 * qb + r;
        const float inv = 1.f / row_sum<D>(acc, qb, r);
        if (qrow >= L) continue;
        const size_t row_off = head_off + (size_t)qrow * D;
#pragma unroll
        for (int mb = 0; mb < G::NDB; ++mb) {
            // no fma contraction: o must be rounded exactly as the parked W was
#pragma clang fp contract(off)
            const int col = 16 * mb + 4 * g;
            if (col >= D) continue;
            const size_t off = row_off + col;
            const f32x4 o = acc.o[qb][mb] * inv;
            f32x4 out = o;
            if constexpr (MODE == MODE_REFRESH) {
                // R is the exact difference of the two rounded fp32 results (a
                // band covering every key gives R == 0 exactly); the window
                // result parked above is read back by the lane that wrote it.
                const f32x4 win = *(const f32x4*)(p.Rout + off);
                *(f32x4*)(p.Rout + off) = o - win;
            }
            if constexpr (MODE == MODE_WINDOW) {
                if (wk.rpre) {
                    // the walk's last iteration left the rows in the stage it freed
                    const float* rl = (const float*)(smem + wk.stage * G::STAGE_ELEMS);
                    out = o + *(const f32x4*)(rl + (qrow - q0) * D + col);
                } else if (p.Rin) {
                    out = o + *(const f32x4*)(p.Rin + off);
                }
            }
            const u32x2 ov = u32x2{pack_bf16x2(out[0], out[1]), pack_bf16x2(out[2], out[3])};
            for (int di = 0; di < p.ndst; ++di) *(u32x2*)(p.dst[di] + off) = ov;
        }
    }
}

// Three waves per SIMD with two query blocks per wavefront (register budget
// 168), four with one (budget 128), three for the two-accumulator refresh: the
// MFMA work of one wavefront overlaps the softmax arithmetic of the others.
template <int QB, int KMODE>
constexpr int waves_per_simd() { return QB == 1 && !split_refresh<KMODE>() ? 4 : 3; }

template <int D, int MODE, int QB>
__global__ void __launch_bounds__(NTHREADS)
    __attribute__((amdgpu_waves_per_eu(waves_per_simd<QB, MODE>(), waves_per_simd<QB, MODE>()))) attn_kernel(Params p) {
    __shared__ __attribute__((aligned(16))) uint16_t smem[2 * Geo<D>::STAGE_ELEMS];
    attn_body<D, MODE, QB>(p, smem);
}

// Streaming copy of n16 16-byte units (AST output reuse).
__global__ void __launch_bounds__(256) copy16_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, size_t n16) {
    const size_t stride = (size_t)gridDim.x * 256 * 4;
    for (size_t base = (size_t)blockIdx.x * 256 * 4 + threadIdx.x; base < n16; base += stride) {
        u32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t i = base + (size_t)u * 256;
            if (i < n16) v[u] = src[i];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t i = base + (size_t)u * 256;
            if (i < n16) dst[i] = v[u];
        }
    }
}

template <int D, int MODE, int QB>
hipError_t launch_attn(const AttnLaunch& a, hipStream_t stream) {
    using G = Geo<D>;
    Params p{};
    p.Q = (const uint16_t*)a.Q;
    p.K = (const uint16_t*)a.K;
    p.V = (const uint16_t*)a.V;
    p.Rin = (const float*)a.Rin;
    p.Rout = (float*)a.Rout;
    p.ndst = a.ndst;
    for (int i = 0; i < 4; ++i) p.dst[i] = (uint16_t*)(i < a.ndst ? a.dst[i] : nullptr);
    p.H = a.H;
    p.L = a.L;
    p.w = a.w;
    p.n_qt = (a.L + bq<QB>() - 1) / bq<QB>();
    const long long nb = (long long)p.n_qt * a.B * a.H;
    if (nb <= 0 || nb > 0x7FFFFFFFLL) return hipErrorInvalidValue;
    p.nblocks = (int)nb;
    p.c = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
    static_assert((size_t)2 * G::STAGE_ELEMS * sizeof(uint16_t) * waves_per_simd<QB, MODE>() <= 160 * 1024,
                  "one workgroup per wave slot of a SIMD must fit in LDS");
    hipLaunchKernelGGL((attn_kernel<D, MODE, QB>), dim3(p.nblocks), dim3(NTHREADS), 0, stream, p);
    return hipGetLastError();
}

// One query block per wavefront (64-query workgroups, four wavefronts per
// SIMD) when a workgroup's tile walk is short: the extra workgroups and
// wavefronts hide latency there.  Long walks run faster with two blocks,
// which halve the K/V tile copies per query.  The crossovers, measured at
// d = 72 with interleaved timings: full attention up to L = 256 (4 key tiles),
// refresh up to L = 1024, window attention up to a band of 1280 keys.  A band
// that covers every key is full attention and takes full attention's choice,
// so that the two give identical results.
template <int MODE>
bool one_query_block(const AttnLaunch& a) {
    // A launch whose 128-query workgroups would number at most one per CU
    // (one wavefront per SIMD) takes 64-query workgroups whatever its length:
    // measured 11% faster at (B, H, L) = (1, 16, 2048) and (4, 16, 512).
    if ((long long)a.B * a.H * ((a.L + bq<2>() - 1) / bq<2>()) <= 256) return true;
    if constexpr (MODE == MODE_REFRESH) return a.L <= 1024;   // L <= 512 takes the split form
    if constexpr (MODE == MODE_WINDOW) {
        if (a.w < a.L - 1) return 2LL * a.w + 1 <= 1280;
    }
    return a.L <= 256;
}

template <int MODE>
hipError_t launch_mode(const AttnLaunch& a, hipStream_t stream) {
    const bool one = one_query_block<MODE>(a);
    switch (a.d) {
        case 64: return one ? launch_attn<64, MODE, 1>(a, stream) : launch_attn<64, MODE, 2>(a, stream);
        case 72: return one ? launch_attn<72, MODE, 1>(a, stream) : launch_attn<72, MODE, 2>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool head_dim_supported(int d) { return d == 64 || d == 72; }

hipError_t launch_full(const AttnLaunch& a, hipStream_t s) { return launch_mode<MODE_FULL>(a, s); }
hipError_t launch_asc(const AttnLaunch& a, hipStream_t s) { return launch_mode<MODE_ASC>(a, s); }
// Refresh: the one-pass two-accumulator form up to L = 512 (8 key tiles, where
// band-edge tiles are most of the walk), the two-phase form beyond (measured:
// L = 256 -16%, 405 -6%, 1024 +3% for the one-pass form).
// Bands of at most 31 keys take the two-phase form with split probabilities
// in its in-band phase (64-query workgroups), so that W, and with it R and
// every reuse that adds R, carries no unaveraged bf16 rounding of its weights.
hipError_t launch_refresh(const AttnLaunch& a, hipStream_t s) {
    if (a.w <= FINE_MAX_HALF_WIDTH && a.w < a.L - 1) {
        switch (a.d) {
            case 64: return launch_attn<64, MODE_REFRESH_FINE, 1>(a, s);
            case 72: return launch_attn<72, MODE_REFRESH_FINE, 1>(a, s);
            default: return hipErrorInvalidValue;
        }
    }
    if (a.L > 512) return launch_mode<MODE_REFRESH>(a, s);
    switch (a.d) {
        case 64: return launch_attn<64, MODE_REFRESH_SPLIT, 1>(a, s);
        case 72: return launch_attn<72, MODE_REFRESH_SPLIT, 1>(a, s);
        default: return hipErrorInvalidValue;
    }
}
// Narrow bands (at most 31 keys per query) apply each probability as a bf16
// value plus its bf16 rounding residual: with so few keys per row the bf16
// rounding of the weights does not average out, and alone it costs up to
// 2^-8 max|v - o| per output.  Such bands always take 64-query workgroups.
// A band covering every key keeps full attention's choice.
hipError_t launch_window(const AttnLaunch& a, hipStream_t s) {
    if (a.w <= FINE_MAX_HALF_WIDTH && a.w < a.L - 1) {
        switch (a.d) {
            case 64: return launch_attn<64, MODE_WINDOW_FINE, 1>(a, s);
            case 72: return launch_attn<72, MODE_WINDOW_FINE, 1>(a, s);
            default: return hipErrorInvalidValue;
        }
    }
    return launch_mode<MODE_WINDOW>(a, s);
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
    const size_t n16 = bytes / 16;
    if (n16 == 0) return hipSuccess;
    size_t blocks = (n16 + 1023) / 1024;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(copy16_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, (const u32x4*)src, (u32x4*)dst, n16);
    return hipGetLastError();
}

}  // namespace dfa
