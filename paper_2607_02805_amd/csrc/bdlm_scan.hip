// bdlm_scan.hip -- gfx950 (CDNA4) kernels for the block-restricted bidirectional
// Mamba scan of BDLM Mamba-H.
//
// What one launch computes, per batch row b and head h (group g = h / (H/G)):
//   forward branch  (Sec. 4, Eq. partial-reverse, first row): the selective
//     update of Sec. 3, Eq. mamba-scan-background, continued through the L block
//     tokens from the cached boundary state s = h_pool[slot(b), h];
//   reverse branch  (second row): the same update over the reversed block from
//     a zero state;
//   y = forward + reverse (third row), written in fp32;
//   commit          (Eq. boundary-state): the forward state after the block
//     replaces s.
//
// Both branches are evaluated in the masked-matrix ("state-space dual") form
// rather than token by token.  With l_t = dt_t A_h, cs_t = l_0 + ... + l_t and
// ex_t = cs_{t-1} (ex_0 = 0):
//   y[t,:] = exp(cs_t) (C_t . s^T)                         prefix (forward only)
//          + sum_j G[t,j] W[t,j] dt_j x[j,:]                both branches at once
//          + (D + D_rev) x[t,:]
//   G[t,j] = C_t . B_j,
//   W[t,j] = exp(cs_t - cs_j)   for j < t   (forward decay from j to t)
//          = 2                  for j = t   (the token's own input, once per branch)
//          = exp(ex_j - ex_t)   for j > t   (reverse decay: a_t ... a_{j-1})
//   s_new  = exp(cs_{L-1}) s + sum_j exp(cs_{L-1} - cs_j) dt_j x[j,:] (outer) B_j
//
// Work decomposition: one workgroup of four 64-wide waves per (b, h); wave w
// owns head-dim columns [16w, 16w+16).  With bf16 activations all contractions run
// on bf16 MFMA (v_mfma_f32_16x16x32_bf16 / 16x16x16) with fp32 accumulation; the
// operands that are not exact in bf16 (the fp32 state and the fp32 decay-weighted
// matrices) are split as v = hi + lo with hi = bf16(v), lo = bf16(v - hi), which
// leaves a relative residual below 2^-16, and products of bf16 values are exact in
// fp32.  With fp32 activations every operand is fp32 and the contractions run on
// fp32 MFMA (v_mfma_f32_16x16x4_f32).
//
// Register layouts.  Every 16x16 MFMA tile uses lane = 16 * grp + col.  An
// operand "quad" is the four values a lane contributes to 16 consecutive
// contraction indices: lane (col, grp) holds indices 4*grp .. 4*grp+3 of that
// run.  Because an MFMA only needs A and B to agree on which contraction index
// each lane slot carries, the state s[p, n] is kept in the accumulator layout
// of the commit product (lane (col = p, grp) holds s[p, 16q + 4grp + r],
// r = 0..3): one 16-byte load per quad q, used directly as the B operand of
// the prefix product and as the accumulator of the commit, then stored back
// with one 16-byte store.  The Gram product is computed transposed (rows j,
// columns t) so that its accumulator is already the A operand of the
// intra-block product.
//
// State layout in HBM: each (slot, head) state is dstate/4 blocks of [64][4]
// floats, s[p, n] at ((n / 4) * 64 + p) * 4 + n % 4.  A wave's 16-byte quad
// loads then cover 1 KB of contiguous memory per instruction.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "bdlm.h"
#include "bdlm_device.h"
#include "bdlm_launch.h"

namespace bdlm {
namespace {

struct KArgs {
    const void *x, *dt, *Bm, *Cm;
    const float *A, *D, *D_rev;
    float *h_pool;
    float *y;
    float *y2;   // kCS: the next block's step outputs
    // kSep: the reverse branch's own inputs (same shapes and strides as the above);
    // kCS: the next block's noised inputs
    const void *x2, *dt2, *Bm2, *Cm2;
    const float *A2;
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int32_t nheads, heads_per_group, L;
    int32_t xcd_remap;   // 1: group consecutive units per XCD (grid % 8 == 0)
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
    // convolution staging: x, B, C are the block's bf16 inputs before the mixer's
    // width-4 depthwise convolution; weights [channels][4], bias [channels], cached
    // last three input rows [slot][3][channels] (fp32)
    const float *conv_w, *conv_b, *conv_pool;
    int32_t conv_ch;
};

// ------------------------------------------------------------------- the kernel
// LT: block tile (16, 32 or 64 tokens; the block length L <= LT, padded tokens
//     have dt = 0, x = B = C = 0, which changes no output and no state).
// NS: dstate.  F32: fp32 activation storage.  COMMIT: also update the state.
// DIR: kBoth computes both branches (one input set for both, Eq. partial-reverse);
//     kFwd only the forward branch from the cached state (skip D) and stores y;
//     kRev only the block-local reverse branch (skip D_rev) and adds it onto y;
//     kCS  commit the clean block (x, dt, B, C; y: its outputs, optional) and then run
//     the next block's first denoising step (x2, dt2, B2, C2, both branches; outputs
//     into y2) from the updated state while it is still in registers: one state read,
//     one state write, the same results as a commit followed by a step;
//     kSep both branches, each from an input set of its own (x, dt, A, B, C for the
//     forward branch, x2, dt2, A2, B2, C2 for the reverse one; bf16 storage, no
//     commit): two Gram matrices, two intra products, one prefix term.  A step whose
//     branches have inputs of their own is one kSep launch, or a kFwd launch followed
//     by a kRev launch on the same stream.
// NPART: the state of a head is split over NPART groups of four waves along
//     dstate (4 * NPART waves per workgroup).  Streaming the state from HBM needs
//     many waves per CU, each with few loads in flight; the partial prefix
//     products of the groups are summed through LDS before y is stored.
//
// Phases:
//   0. every global load is issued unconditionally (rows past the block read a
//      zero chunk): B, C, x, dt and the per-head parameters in coalesced 16-byte
//      chunks by the whole workgroup, then the first half of this wave's share of
//      the state, 16 bytes per quad, into registers (the second half follows the
//      first barrier);
//   1. B and C are written to LDS as "register images" (the exact per-lane quads
//      an MFMA operand needs, so reading one is a linear, conflict-free 8-byte
//      read), x row-major; wave 0 runs the decay prefix sums of the block on DPP
//      (lane t = token t) and publishes dt, cs and ex as floats;
//   2. the Gram tiles are shared out over the waves, turned into the
//      decay-weighted matrix M[t,j] = G[t,j] W[t,j] dt_j, split and published in
//      LDS;
//   3. the first group contracts M with x (its 16 columns) and precomputes the
//      skip term and the prefix scales; every wave contracts C with its rows and
//      dstate quads of the state (the only step that waits for the state loads);
//      the partial products are summed and y is stored; a commit then adds the
//      block to each wave's quads of the state in place.
constexpr int kBoth = 0, kFwd = 1, kRev = 2, kSep = 3, kCS = 4;

// c += a b over one quad of 16 contraction indices on fp32 MFMA: instruction r takes
// value r of every lane, i.e. index 4 grp + r of the quad layout.
__device__ __forceinline__ f32x4 mma_q32(f32x4 a, f32x4 b, f32x4 c) {
#pragma unroll
    for (int r = 0; r < 4; ++r) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[r], b[r], c, 0, 0, 0);
    return c;
}

// One 16 x 16 tile of the decay-weighted matrix M[t, j] = G[t, j] W[t, j] dt_j from bf16
// operand images (rows t of token tile mt, columns j of token tile jt), held transposed
// (lane (grp, col): j = 16 jt + 4 grp + r, t = 16 mt + col) and split into bf16 hi (xy)
// and lo (zw).  WDIR selects the weights: kBoth both triangles and 2 on the diagonal,
// kFwd the lower triangle, kRev the upper one (1 on the diagonal).
template <int QN, int WDIR>
__device__ __forceinline__ uint4 gram_tile_bf16(const uint2 *iB, const uint2 *iC, const float *dCs,
                                                const float *dEx, const float *dDt, int mt, int jt,
                                                int grp, int col) {
    // accumulator holds G[t, j] for t = 16mt + col, j = 16jt + 4grp + r
    f32x4 gacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < QN; q += 2) {   // two dstate quads per product
        const int q1 = q + 1 < QN ? q + 1 : q;
        const s16x4 b0 = as_s16x4(iB[img_idx<QN, false>(jt, q, grp, col)]);
        const s16x4 b1 = as_s16x4(iB[img_idx<QN, false>(jt, q1, grp, col)]);
        const s16x4 c0 = as_s16x4(iC[img_idx<QN, false>(mt, q, grp, col)]);
        const s16x4 c1 = as_s16x4(iC[img_idx<QN, false>(mt, q1, grp, col)]);
        if (q + 1 < QN) gacc = mma_k32(b0, b1, c0, c1, gacc);
        else gacc = mma_k16(b0, c0, gacc);
    }
    const int t = 16 * mt + col;
    const float cst = dCs[t], ext = dEx[t];
    const f32x4 csj = *reinterpret_cast<const f32x4 *>(&dCs[16 * jt + 4 * grp]);
    const f32x4 exj = *reinterpret_cast<const f32x4 *>(&dEx[16 * jt + 4 * grp]);
    const f32x4 dtj = *reinterpret_cast<const f32x4 *>(&dDt[16 * jt + 4 * grp]);
    f32x4 m;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        // below the diagonal the forward decay from j to t, above it the reverse decay
        // a_t ... a_{j-1}; on it the token's own input, once per branch computed here
        const int j = 16 * jt + 4 * grp + r;
        const float e = exp2f(j < t ? cst - csj[r] : exj[r] - ext);
        const float w = j == t ? (WDIR == kBoth ? 2.f : 1.f)
                               : (j < t ? (WDIR == kRev ? 0.f : e) : (WDIR == kFwd ? 0.f : e));
        m[r] = gacc[r] * w * dtj[r];
    }
    s16x4 mh, ml;
    split4(m, mh, ml);
    const uint2 a = as_u2(mh), c2 = as_u2(ml);
    return uint4{a.x, a.y, c2.x, c2.y};
}

// The same tile from fp32 operand images on fp32 MFMA, unsplit (fp32 storage).
template <int QN, int WDIR>
__device__ __forceinline__ uint4 gram_tile_f32(const f32x4 *iB, const f32x4 *iC, const float *dCs,
                                               const float *dEx, const float *dDt, int mt, int jt,
                                               int grp, int col) {
    f32x4 gacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < QN; ++q)
        gacc = mma_q32(iB[img_idx<QN, true>(jt, q, grp, col)], iC[img_idx<QN, true>(mt, q, grp, col)], gacc);
    const int t = 16 * mt + col;
    const float cst = dCs[t], ext = dEx[t];
    const f32x4 csj = *reinterpret_cast<const f32x4 *>(&dCs[16 * jt + 4 * grp]);
    const f32x4 exj = *reinterpret_cast<const f32x4 *>(&dEx[16 * jt + 4 * grp]);
    const f32x4 dtj = *reinterpret_cast<const f32x4 *>(&dDt[16 * jt + 4 * grp]);
    f32x4 m;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int j = 16 * jt + 4 * grp + r;
        const float e = exp2f(j < t ? cst - csj[r] : exj[r] - ext);
        const float w = j == t ? (WDIR == kBoth ? 2.f : 1.f)
                               : (j < t ? (WDIR == kRev ? 0.f : e) : (WDIR == kFwd ? 0.f : e));
        m[r] = gacc[r] * w * dtj[r];
    }
    return __builtin_bit_cast(uint4, m);
}

// CV: the block's x, B and C are convolved while they are staged (bf16 inputs before
// the mixer's convolution, fp32 operands after it; forward: the convolution continues
// from the cached rows, reverse: zero past the block's end).
template <int LT, int NS, bool F32, bool COMMIT, int NPART, int DIR, bool CV>
__global__ void __launch_bounds__(256 * NPART)
__attribute__((amdgpu_waves_per_eu(2 * NPART)))
bdlm_block_kernel(const KArgs args) {
    static_assert(DIR == kBoth || DIR == kFwd || DIR == kRev || DIR == kSep || DIR == kCS,
                  "direction");
    static_assert(DIR != kCS || (!F32 && COMMIT && !CV), "commit + step: bf16 storage");
    static_assert(!CV || (F32 && (DIR == kFwd || DIR == kRev || DIR == kSep) && LT <= 32),
                  "convolution staging");
    static_assert(!(COMMIT && DIR == kRev), "a commit updates the forward state");
    constexpr bool SEP = DIR == kSep;
    constexpr bool TWO = SEP || DIR == kCS;   // a second input set is staged
    // separate input sets: bf16 storage and steps only, except under convolution staging,
    // where the two sets are the block's forward and reverse convolutions (fp32, and a
    // commit updates the state from the forward set)
    static_assert(!(SEP && !CV && (F32 || COMMIT)), "separate inputs: bf16 storage, step only");
    constexpr int NT = 256 * NPART;       // threads
    constexpr int NW = 4 * NPART;         // waves
    constexpr int MT = LT / 16;           // token tiles = quads along the block
    constexpr int QN = NS / 16;           // quads along dstate
    constexpr int QW = QN / NPART;        // dstate quads per wave
    static_assert(QN % NPART == 0 && QW >= 1, "dstate split");
    constexpr int IMG = MT * QN * 64;     // quads in one image of B or C
    constexpr int E = F32 ? 4 : 8;        // activations per 16-byte chunk
    constexpr int XS = kP + 4;            // x row stride in LDS (elements)
    using AT = typename Act<F32>::T;

    // operand images of C and B: bf16 quads, or fp32 quads for fp32 storage (fp32
    // activations are contracted on fp32 MFMA: all-fp32 operands lose too much to
    // cancellation under two-term bf16 splits)
    __shared__ __align__(16) uint2 sC[F32 ? 1 : IMG], sB[F32 ? 1 : IMG];
    __shared__ __align__(16) f32x4 sCf[F32 ? IMG : 1], sBf[F32 ? IMG : 1];
    __shared__ __align__(16) AT sX[LT * XS];
    using DT = typename Act<F32 && !CV>::T;   // dt storage (bf16 under convolution staging)
    __shared__ __align__(16) float sDt[64], sCs[64], sEx[64];   // dt, cs, ex per token
    __shared__ float sPar[4];                                          // A[h], D[h], D_rev[h]
    __shared__ __align__(16) uint4 sM[MT * MT * 64];                  // M: hi (xy), lo (zw)
    // the second input set's images, x, decay sums and matrix (kSep: the reverse branch;
    // kCS: the next block)
    __shared__ __align__(16) uint2 sC2[TWO && !F32 ? IMG : 1], sB2[TWO && !F32 ? IMG : 1];
    // (the block's reverse convolution, CV, passes through sBf / sCf before the forward one)
    __shared__ __align__(16) f32x4 sCf2[TWO && F32 && !CV ? IMG : 1], sBf2[TWO && F32 && !CV ? IMG : 1];
    __shared__ __align__(16) AT sX2[TWO ? LT * XS : 1];
    __shared__ __align__(16) float sDt2[TWO && !CV ? 64 : 1], sCs2[TWO && !CV ? 64 : 1],
        sEx2[TWO && !CV ? 64 : 1];
    __shared__ __align__(16) uint4 sM2[TWO ? MT * MT * 64 : 1];
    __shared__ __align__(16) f32x4 sRed[(NPART > 1 ? NPART - 1 : 1) * 4 * MT * 64];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int pblk = wave & 3, part = wave >> 2;   // 16 head-dim columns, dstate share
    const int col = lane & 15, grp = lane >> 4;

    // Unit (b, h).  Workgroups are dealt to the 8 XCDs round-robin; remapping
    // gives each XCD a contiguous run of units, so the heads of one batch row
    // (which share B and C) sit behind one L2.
    int u = blockIdx.x;
    if (args.xcd_remap) u = (u & 7) * (static_cast<int>(gridDim.x) >> 3) + (u >> 3);
    const int b = u / args.nheads;
    const int h = u - b * args.nheads;
    const int g = h / args.heads_per_group;
    const int64_t slot = args.use_slots ? args.slots[b] : b;
    const int L = args.L;                 // 1 <= L <= LT
    const int p = pblk * 16 + col;
    const int q0 = part * QW;             // first dstate quad of this wave

    const AT *xg = static_cast<const AT *>(args.x) + b * args.xs_b + h * args.xs_h;
    const DT *dtg = static_cast<const DT *>(args.dt) + b * args.dts_b + h;
    const AT *Bg = static_cast<const AT *>(args.Bm) + b * args.bcs_b + g * args.bcs_g;
    const AT *Cg = static_cast<const AT *>(args.Cm) + b * args.bcs_b + g * args.bcs_g;
    // this lane's quads of the state: s[p, 16q + 4grp + r] at hs + q * 1024
    float *hs = args.h_pool + (slot * args.nheads + h) * kP * NS + (grp * kP + p) * 4;

    // ---- phase 0: loads
    constexpr int CPR = NS / E;                           // 16-byte chunks per row
    constexpr int BC_CH = LT * CPR;                       // chunks per matrix
    // Chunk counts are multiples of 64 (or below 64, then one partial wave loads
    // them), so "this thread owns chunk i" is decided per wave.
    constexpr int BC_PT = BC_CH >= NT ? BC_CH / NT : 1;
    const bool bc_owner = tid < BC_CH;
    u32x4 cch[BC_PT], bch[BC_PT];
    if (!CV && bc_owner) {
#pragma unroll
        for (int k = 0; k < BC_PT; ++k) {
            const int i = tid + NT * k;                    // chunk fastest (coalesced)
            const int t = i / CPR, c = i % CPR;
            const int64_t o = t * args.bcs_t + c * E;
            const bool ok = t < L;
            cch[k] = __builtin_nontemporal_load(ok ? gchunk(Cg + o) : gzero());
            bch[k] = __builtin_nontemporal_load(ok ? gchunk(Bg + o) : gzero());
        }
    }
    constexpr int X_CH = LT * (kP / E);
    constexpr int X_PT = X_CH >= NT ? X_CH / NT : 1;
    const bool x_owner = tid < X_CH;
    u32x4 xch[X_PT];
    if (!CV && x_owner) {
#pragma unroll
        for (int k = 0; k < X_PT; ++k) {
            const int i = tid + NT * k;                    // chunk fastest (coalesced)
            const int j = i / (kP / E), c = i % (kP / E);
            xch[k] = __builtin_nontemporal_load(j < L ? gchunk(xg + j * args.xs_t + c * E)
                                                      : gzero());
        }
    }
    u32x4 cch2[TWO ? BC_PT : 1], bch2[TWO ? BC_PT : 1], xch2[TWO ? X_PT : 1];
    if constexpr (TWO && !CV) {
        const AT *Bg2 = static_cast<const AT *>(args.Bm2) + b * args.bcs_b + g * args.bcs_g;
        const AT *Cg2 = static_cast<const AT *>(args.Cm2) + b * args.bcs_b + g * args.bcs_g;
        const AT *xg2 = static_cast<const AT *>(args.x2) + b * args.xs_b + h * args.xs_h;
        if (bc_owner) {
#pragma unroll
            for (int k = 0; k < BC_PT; ++k) {
                const int i = tid + NT * k;
                const int t = i / CPR, c = i % CPR;
                const int64_t o = t * args.bcs_t + c * E;
                const bool ok = t < L;
                cch2[k] = __builtin_nontemporal_load(ok ? gchunk(Cg2 + o) : gzero());
                bch2[k] = __builtin_nontemporal_load(ok ? gchunk(Bg2 + o) : gzero());
            }
        }
        if (x_owner) {
#pragma unroll
            for (int k = 0; k < X_PT; ++k) {
                const int i = tid + NT * k;
                const int j = i / (kP / E), c = i % (kP / E);
                xch2[k] = __builtin_nontemporal_load(j < L ? gchunk(xg2 + j * args.xs_t + c * E)
                                                           : gzero());
            }
        }
    }
    // dt (lane t = token t), loaded by every wave though wave 0 alone stages it: where
    // a load under a branch joins the other path the compiler converts its value right
    // away, i.e. waits there for every load issued before it (the state loads of wave 0
    // would then leave only after all of its inputs had arrived)
    typedef __attribute__((address_space(1))) const AT g_at;
    typedef __attribute__((address_space(1))) const DT g_dt;
    const DT dtraw = *(lane < L ? (const g_dt *)(dtg + lane * args.dts_t)
                                : (const g_dt *)(&kZeroChunk));
    DT dtraw2 = DT(0);
    if constexpr (TWO) {
        const DT *dtg2 = static_cast<const DT *>(args.dt2) + b * args.dts_b + h;
        dtraw2 = *(lane < L ? (const g_dt *)(dtg2 + lane * args.dts_t) : (const g_dt *)(&kZeroChunk));
    }
    // per-head parameters as vector loads in this first batch: a scalar load issued
    // later would queue behind the state loads of every workgroup
    typedef __attribute__((address_space(1))) const float g_f;
    float parv = 0.f;
    if (wave == 0) {
        const float *par = tid == 0 ? args.A
                                    : (tid == 1 ? args.D : (SEP && tid == 3 ? args.A2 : args.D_rev));
        parv = *(const g_f *)(par + h);
    }
    // Convolution staging: task (matrix, channel quad, 8-token group) loads the input rows
    // its 8 outputs need (each row the sum of a cached-row load and an input-row load, the
    // one that does not apply reading a zero chunk), the 4 channels' weights and biases:
    // rows t0-3 .. t0+7 for the forward convolution (before the block: the cache), t0 ..
    // t0+10 for the reverse one (zero past the block's end), t0-3 .. t0+10 for both (kSep:
    // the first input set is the forward convolution, the second the reverse one).
    constexpr int CQX = kP / 4, CQB = NS / 4, TG = LT / 8;
    constexpr int CV_TASKS = (CQX + 2 * CQB) * TG;
    static_assert(!CV || CV_TASKS <= NT, "one convolution task per thread");
    constexpr int CV_ROWS = DIR == kSep ? 14 : 11;
    constexpr int CV_BASE = DIR == kRev ? 0 : 3;   // row i of the task is token t0 - CV_BASE + i
    f32x4 cu[CV ? CV_ROWS : 1], cw[CV ? 4 : 1], cb = {0.f, 0.f, 0.f, 0.f};
    int cv_m = 0, cv_q = 0, cv_t0 = 0;   // matrix (0 x, 1 B, 2 C), channel quad, first token
    if constexpr (CV) {
        typedef unsigned v2u __attribute__((ext_vector_type(2)));
        typedef __attribute__((address_space(1))) const f32x4 g_f4;
        typedef __attribute__((address_space(1))) const v2u g_u2;
        const int task = tid < CV_TASKS ? tid : 0;   // threads past the tasks repeat task 0
        const int per_tg = CQX + 2 * CQB;
        cv_t0 = 8 * (task / per_tg);
        const int r = task % per_tg;
        cv_m = r < CQX ? 0 : (r < CQX + CQB ? 1 : 2);
        cv_q = r < CQX ? r : (r < CQX + CQB ? r - CQX : r - CQX - CQB);
        const int HP = args.nheads * kP, GN = (args.nheads / args.heads_per_group) * NS;
        const int c = cv_m == 0 ? h * kP + 4 * cv_q : HP + (cv_m - 1) * GN + g * NS + 4 * cv_q;
        const uint16_t *src = static_cast<const uint16_t *>(cv_m == 0 ? args.x : (cv_m == 1 ? args.Bm : args.Cm)) +
                              b * (cv_m == 0 ? args.xs_b : args.bcs_b) +
                              (cv_m == 0 ? h * args.xs_h : g * args.bcs_g) + 4 * cv_q;
        const int64_t rs = cv_m == 0 ? args.xs_t : args.bcs_t;
        const float *crow = args.conv_pool + slot * 3 * static_cast<int64_t>(args.conv_ch) + c;
#pragma unroll
        for (int i = 0; i < CV_ROWS; ++i) {
            const int rr = cv_t0 - CV_BASE + i;
            const bool in_blk = rr >= 0 && rr < L;
            const v2u u = *(in_blk ? (const g_u2 *)(src + rr * rs) : (const g_u2 *)(&kZeroChunk));
            f32x4 v = f32x4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                            __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
            if constexpr (DIR != kRev)
                v += *(rr < 0 ? (const g_f4 *)(crow + (rr < 0 ? rr + 3 : 0) * args.conv_ch)
                              : (const g_f4 *)(&kZeroChunk));
            cu[i] = v;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) cw[e] = *(const g_f4 *)(args.conv_w + 4 * static_cast<int64_t>(c + e));
        cb = *(const g_f4 *)(args.conv_b + c);
    }
    // keep the small loads above ahead of the state loads (loads return in order)
    __builtin_amdgcn_sched_barrier(0);
    // The state is requested in two halves: the first now, the second once the
    // workgroup's inputs have arrived (after the first barrier).  With every state
    // load of the chip in flight at once, the input loads of a workgroup queue behind
    // them and hold up all the work that does not need the state; the second half
    // still arrives before it is needed.  Everything here is read once per step and
    // streams past the caches (nontemporal).
    constexpr int QE = (QW + 1) / 2;   // state quads requested up front
    f32x4 hq[QW];  // state s[p, 16(q0 + k) + 4grp + r]
    auto load_state = [&](int k) {
        if constexpr (DIR == kRev) hq[k] = f32x4{0.f, 0.f, 0.f, 0.f};   // the state is not used
        else hq[k] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(hs + (q0 + k) * 16 * kP));
    };
#pragma unroll
    for (int k = 0; k < QE; ++k) load_state(k);

    // ---- phase 1: LDS images
    // one direction's 8 outputs of the task, convolved and through SiLU, into (dX, dB,
    // dC): forward w0 u[t-3] + ... + w3 u[t], reverse w0 u[t+3] + ... + w3 u[t]
    auto conv_emit = [&](auto rev_tag, AT *dX, f32x4 *dB, f32x4 *dC) {
        constexpr bool rev = decltype(rev_tag)::value;   // a template: instantiated only under CV
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int t = cv_t0 + i;
            f32x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float a = cb[e];
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    a += cw[e][k] * cu[rev ? i + 3 + CV_BASE - k : i + k + CV_BASE - 3][e];
                // SiLU a / (1 + e^-a) on the hardware exp2 and reciprocal (each within
                // a few ulp; the B and C channels are convolved by every head's
                // workgroup, so this runs 5x more often than one pass over the
                // channels); padded rows stay zero
                const float sg = __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-a * kLog2e));
                o[e] = t < L ? a * sg : 0.f;
            }
            if (cv_m == 0) {
                *reinterpret_cast<f32x4 *>(&dX[t * XS + 4 * cv_q]) = o;
            } else {
                const int at = img_idx<QN, true>(t >> 4, cv_q >> 2, cv_q & 3, t & 15);
                if (cv_m == 1) dB[at] = o;
                else dC[at] = o;
            }
        }
    };
    if constexpr (CV) {
        // both directions (kSep): the reverse convolution first, through the same images
        // as the forward one; its Gram tiles are formed and kept (below) before the forward
        // convolution overwrites them, so two fp32 image sets fit in the LDS of one
        if (tid < CV_TASKS) {
            if constexpr (DIR == kSep) conv_emit(std::true_type{}, sX2, sBf, sCf);
            else conv_emit(std::integral_constant<bool, DIR == kRev>{}, sX, sBf, sCf);
        }
    }
#pragma unroll
    for (int k = 0; k < BC_PT; ++k) {
        if (CV || !bc_owner) break;
        const int i = tid + NT * k;
        const int t = i / CPR, c = i % CPR;
        const u32x4 cz = cch[k], bz = bch[k];
        if constexpr (F32) {
            // 4 floats = one quad: q = c / 4, grp = c % 4
            const int at = img_idx<QN, F32>(t >> 4, c >> 2, c & 3, t & 15);
            sCf[at] = __builtin_bit_cast(f32x4, cz);
            sBf[at] = __builtin_bit_cast(f32x4, bz);
        } else {
            // 8 bf16 = two quads: q = c / 2, grp = 2 (c % 2) and 2 (c % 2) + 1
            const int at = img_idx<QN, F32>(t >> 4, c >> 1, 2 * (c & 1), t & 15);
            sC[at] = uint2{cz.x, cz.y};
            sC[at + 16] = uint2{cz.z, cz.w};
            sB[at] = uint2{bz.x, bz.y};
            sB[at + 16] = uint2{bz.z, bz.w};
        }
    }
#pragma unroll
    for (int k = 0; k < X_PT; ++k) {
        if (CV || !x_owner) break;
        const int i = tid + NT * k;
        const int j = i / (kP / E), c = i % (kP / E);
        const u32x4 v = xch[k];
        uint2 *dst = reinterpret_cast<uint2 *>(&sX[j * XS + c * E]);
        dst[0] = uint2{v.x, v.y};
        dst[1] = uint2{v.z, v.w};
    }
    if constexpr (TWO) {
#pragma unroll
        for (int k = 0; k < BC_PT; ++k) {
            if (CV || !bc_owner) break;
            const int i = tid + NT * k;
            const int t = i / CPR, c = i % CPR;
            const u32x4 cz = cch2[k], bz = bch2[k];
            const int at = img_idx<QN, false>(t >> 4, c >> 1, 2 * (c & 1), t & 15);
            sC2[at] = uint2{cz.x, cz.y};
            sC2[at + 16] = uint2{cz.z, cz.w};
            sB2[at] = uint2{bz.x, bz.y};
            sB2[at + 16] = uint2{bz.z, bz.w};
        }
#pragma unroll
        for (int k = 0; k < X_PT; ++k) {
            if (CV || !x_owner) break;
            const int i = tid + NT * k;
            const int j = i / (kP / E), c = i % (kP / E);
            const u32x4 v = xch2[k];
            uint2 *dst = reinterpret_cast<uint2 *>(&sX2[j * XS + c * E]);
            dst[0] = uint2{v.x, v.y};
            dst[1] = uint2{v.z, v.w};
        }
        if (SEP && tid == 3) sPar[3] = parv;   // A of the reverse branch
    }
    if (tid < 3) sPar[tid] = parv;
    if (wave == 0) {
        // decay sums of the block in base 2 (lane t = token t; padded tokens have dt = 0):
        // cs_t = l_0 + ... + l_t with l_t = dt_t A_h, and ex_t = cs_{t-1} (ex_0 = 0)
        const float dtv = Act<F32 && !CV>::val(dtraw);
        const float A2 =
            __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(parv))) * kLog2e;
        const float cs = wave_inclusive_sum(dtv * A2);
        const float up = __shfl_up(cs, 1, 64);
        sDt[lane] = dtv;
        sCs[lane] = cs;
        sEx[lane] = lane == 0 ? 0.f : up;
        if constexpr (TWO && !CV) {   // the second set's decay sums (kSep: its own dt and A)
            const float dtv2 = Act<F32 && !CV>::val(dtraw2);
            const float Ar2 =
                __int_as_float(__builtin_amdgcn_readlane(__float_as_int(parv), SEP ? 3 : 0)) *
                kLog2e;
            const float cs2 = wave_inclusive_sum(dtv2 * Ar2);
            const float up2 = __shfl_up(cs2, 1, 64);
            sDt2[lane] = dtv2;
            sCs2[lane] = cs2;
            sEx2[lane] = lane == 0 ? 0.f : up2;
        }
    }
    if constexpr (CV && SEP) {
        __syncthreads();   // the reverse convolution's images and the decay sums
        for (int tile = wave; tile < MT * MT; tile += NW)
            sM2[tile * 64 + lane] =
                gram_tile_f32<QN, kRev>(sBf, sCf, sCs, sEx, sDt, tile / MT, tile % MT, grp, col);
        __syncthreads();   // its tiles are formed: the images are overwritten next
        if (tid < CV_TASKS) conv_emit(std::false_type{}, sX, sBf, sCf);
    }
    __syncthreads();
#pragma unroll
    for (int k = QE; k < QW; ++k) load_state(k);

    // ---- phase 2: Gram tiles (shared out)

    if constexpr (DIR == kCS) {
        // the clean block's tiles (only for its outputs), then the next block's
        const int n1 = args.y != nullptr ? MT * MT : 0;
        for (int tile = wave; tile < n1 + MT * MT; tile += NW) {
            if (tile < n1)
                sM[tile * 64 + lane] = gram_tile_bf16<QN, kBoth>(sB, sC, sCs, sEx, sDt, tile / MT,
                                                                 tile % MT, grp, col);
            else
                sM2[(tile - n1) * 64 + lane] = gram_tile_bf16<QN, kBoth>(
                    sB2, sC2, sCs2, sEx2, sDt2, (tile - n1) / MT, (tile - n1) % MT, grp, col);
        }
    } else if constexpr (SEP) {
        // forward tiles from the first input set, reverse tiles from the second
        for (int tile = wave; tile < 2 * MT * MT; tile += NW) {
            const int tt = tile < MT * MT ? tile : tile - MT * MT;
            const int mt = tt / MT, jt = tt % MT;
            if constexpr (F32) {   // the block's two convolutions: the reverse tiles are formed
                if (tile < MT * MT)  // while staging, only the forward ones here
                    sM[tt * 64 + lane] = gram_tile_f32<QN, kFwd>(sBf, sCf, sCs, sEx, sDt, mt, jt, grp, col);
            } else {
                if (tile < MT * MT)
                    sM[tt * 64 + lane] = gram_tile_bf16<QN, kFwd>(sB, sC, sCs, sEx, sDt, mt, jt, grp, col);
                else
                    sM2[tt * 64 + lane] = gram_tile_bf16<QN, kRev>(sB2, sC2, sCs2, sEx2, sDt2, mt, jt, grp, col);
            }
        }
    } else if constexpr (!F32) {
        for (int tile = wave; tile < MT * MT; tile += NW)
            sM[tile * 64 + lane] =
                gram_tile_bf16<QN, DIR>(sB, sC, sCs, sEx, sDt, tile / MT, tile % MT, grp, col);
    } else {   // fp32 storage: fp32 MFMA, fp32 matrix
        for (int tile = wave; tile < MT * MT; tile += NW) {
            const int mt = tile / MT, jt = tile % MT;
            // accumulator holds G[t, j] for t = 16mt + col, j = 16jt + 4grp + r
            f32x4 gacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < QN; ++q)
                gacc = mma_q32(sBf[img_idx<QN, F32>(jt, q, grp, col)],
                               sCf[img_idx<QN, F32>(mt, q, grp, col)], gacc);
            const int t = 16 * mt + col;
            const float cst = sCs[t], ext = sEx[t];
            const f32x4 csj = *reinterpret_cast<const f32x4 *>(&sCs[16 * jt + 4 * grp]);
            const f32x4 exj = *reinterpret_cast<const f32x4 *>(&sEx[16 * jt + 4 * grp]);
            const f32x4 dtj = *reinterpret_cast<const f32x4 *>(&sDt[16 * jt + 4 * grp]);
            f32x4 m;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                // below the diagonal the forward decay from j to t, above it the reverse decay
                // a_t ... a_{j-1}; on it the token's own input, once per branch computed here
                const int j = 16 * jt + 4 * grp + r;
                const float e = exp2f(j < t ? cst - csj[r] : exj[r] - ext);
                const float w = j == t ? (DIR == kBoth ? 2.f : 1.f)
                                       : (j < t ? (DIR == kRev ? 0.f : e) : (DIR == kFwd ? 0.f : e));
                m[r] = gacc[r] * w * dtj[r];
            }
            sM[tile * 64 + lane] = __builtin_bit_cast(uint4, m);
        }
    }
    __syncthreads();

    // ---- phase 3: x quads (B operand, j = 16jt + 4grp + r), products, output
    float xv[MT][4];
    s16x4 xq[MT];   // bf16 storage: the x quads are exact in bf16
#pragma unroll
    for (int jt = 0; jt < MT; ++jt) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
            xv[jt][r] = Act<F32>::val(sX[(16 * jt + 4 * grp + r) * XS + p]);
        if constexpr (!F32) {
            s16x4 lo;
            split4(f32x4{xv[jt][0], xv[jt][1], xv[jt][2], xv[jt][3]}, xq[jt], lo);
        }
    }
    auto xquad = [&](int jt) { return f32x4{xv[jt][0], xv[jt][1], xv[jt][2], xv[jt][3]}; };
    float xv2[TWO ? MT : 1][4];
    s16x4 xq2[TWO ? MT : 1];
    if constexpr (TWO) {
#pragma unroll
        for (int jt = 0; jt < MT; ++jt) {
#pragma unroll
            for (int r = 0; r < 4; ++r) xv2[jt][r] = Act<F32>::val(sX2[(16 * jt + 4 * grp + r) * XS + p]);
            s16x4 lo;
            split4(f32x4{xv2[jt][0], xv2[jt][1], xv2[jt][2], xv2[jt][3]}, xq2[jt], lo);
        }
    }

    float *yb = args.y;
    const bool want_y = !COMMIT || yb != nullptr;
    if (want_y) {
        // first group: intra-block product, skip term and prefix scales, all before
        // waiting for the state
        float pre[MT][4], es[MT][4];
        if (part == 0) {
            const float skip = DIR == kBoth || DIR == kCS ? sPar[1] + sPar[2]
                                                           : (DIR == kFwd || SEP ? sPar[1] : sPar[2]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                f32x4 ai = {0.f, 0.f, 0.f, 0.f};
                if constexpr (F32) {
#pragma unroll
                    for (int jt = 0; jt < MT; ++jt)
                        ai = mma_q32(__builtin_bit_cast(f32x4, sM[(mt * MT + jt) * 64 + lane]),
                                     xquad(jt), ai);
                    if constexpr (SEP) {   // + the reverse convolution's intra product and skip
#pragma unroll
                        for (int jt = 0; jt < MT; ++jt)
                            ai = mma_q32(__builtin_bit_cast(f32x4, sM2[(mt * MT + jt) * 64 + lane]),
                                         f32x4{xv2[jt][0], xv2[jt][1], xv2[jt][2], xv2[jt][3]}, ai);
#pragma unroll
                        for (int r = 0; r < 4; ++r) ai[r] += sPar[2] * xv2[mt][r];
                    }
                } else {
                    s16x4 mh[MT], ml[MT];
#pragma unroll
                    for (int jt = 0; jt < MT; ++jt) {
                        const uint4 v = sM[(mt * MT + jt) * 64 + lane];
                        mh[jt] = as_s16x4(uint2{v.x, v.y});
                        ml[jt] = as_s16x4(uint2{v.z, v.w});
                    }
                    ai = mma_quads<MT>(mh, xq, ai);
                    ai = mma_quads<MT>(ml, xq, ai);
                    if constexpr (SEP) {   // + the reverse branch's intra product and skip
#pragma unroll
                        for (int jt = 0; jt < MT; ++jt) {
                            const uint4 v = sM2[(mt * MT + jt) * 64 + lane];
                            mh[jt] = as_s16x4(uint2{v.x, v.y});
                            ml[jt] = as_s16x4(uint2{v.z, v.w});
                        }
                        ai = mma_quads<MT>(mh, xq2, ai);
                        ai = mma_quads<MT>(ml, xq2, ai);
#pragma unroll
                        for (int r = 0; r < 4; ++r) ai[r] += sPar[2] * xv2[mt][r];
                    }
                }
                const f32x4 csq = *reinterpret_cast<const f32x4 *>(&sCs[16 * mt + 4 * grp]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    pre[mt][r] = ai[r] + skip * xv[mt][r];
                    es[mt][r] = exp2f(csq[r]);
                    pin(pre[mt][r]);
                    pin(es[mt][r]);
                }
            }
        }
        // C quads of this wave's dstate share, before the state wait
        s16x4 cq[MT][F32 ? 1 : QW];
        f32x4 cf[MT][F32 ? QW : 1];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int k = 0; k < QW; ++k) {
                if constexpr (F32) cf[mt][k] = sCf[img_idx<QN, F32>(mt, q0 + k, grp, col)];
                else cq[mt][k] = as_s16x4(sC[img_idx<QN, F32>(mt, q0 + k, grp, col)]);
            }
        __builtin_amdgcn_sched_barrier(0);   // keep the above ahead of the state wait

        // partial prefix term: C (rows t) against this wave's state quads (columns
        // p), a pair of quads at a time as the loads return
        f32x4 ap[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) ap[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (F32) {
#pragma unroll
            for (int k = 0; k < (DIR == kRev ? 0 : QW); ++k)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) ap[mt] = mma_q32(cf[mt][k], hq[k], ap[mt]);
        } else {
#pragma unroll
            for (int k = 0; k < (DIR == kRev ? 0 : QW); k += 2) {
                if (k + 1 < QW) {
                    s16x4 h0, l0, h1, l1;
                    split4(hq[k], h0, l0);
                    split4(hq[k + 1], h1, l1);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        ap[mt] = mma_k32(cq[mt][k], cq[mt][k + 1], h0, h1, ap[mt]);
                        ap[mt] = mma_k32(cq[mt][k], cq[mt][k + 1], l0, l1, ap[mt]);
                    }
                } else {
                    s16x4 h0, l0;
                    split4(hq[k], h0, l0);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        ap[mt] = mma_k16(cq[mt][k], h0, ap[mt]);
                        ap[mt] = mma_k16(cq[mt][k], l0, ap[mt]);
                    }
                }
            }
        }
        if constexpr (NPART > 1 && DIR != kRev) {
            if (part > 0)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    sRed[(((part - 1) * 4 + pblk) * MT + mt) * 64 + lane] = ap[mt];
            __syncthreads();
            if (part == 0)
#pragma unroll
                for (int pt = 1; pt < NPART; ++pt)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        ap[mt] += sRed[(((pt - 1) * 4 + pblk) * MT + mt) * 64 + lane];
        }
        if (part == 0) {
            // y straight from the accumulators: lanes of a group write 64 contiguous bytes
            float *yrow = yb + ((static_cast<int64_t>(b) * L + 4 * grp) * args.nheads + h) * kP + p;
            const int ytok = args.nheads * kP;           // elements between consecutive tokens
            if constexpr (DIR == kRev) {
                // add onto the forward launch's outputs (one writer per element)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (16 * mt + 4 * grp + r < L) {
                            float *at = yrow + (16 * mt + r) * ytok;
                            __builtin_nontemporal_store(*at + pre[mt][r], at);
                        }
            } else if (L == LT) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        __builtin_nontemporal_store(es[mt][r] * ap[mt][r] + pre[mt][r],
                                                    yrow + (16 * mt + r) * ytok);
            } else {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (16 * mt + 4 * grp + r < L)
                            __builtin_nontemporal_store(es[mt][r] * ap[mt][r] + pre[mt][r],
                                                        yrow + (16 * mt + r) * ytok);
            }
        }
    }

    if constexpr (COMMIT) {
        // s_new[p, n] = exp(cs_last) s[p, n] + sum_j x[j, p] exp(cs_last - cs_j) dt_j B[j, n]
        // on this wave's dstate quads.  A operand: lane (col, grp) holds the weighted
        // B[16jt + 4grp + r, 16q + col], read from the B image (element (j, n) sits in
        // the quad of tile j/16, quad n/16, group n%16/4, column j%16, at slot n%4).
        const float cl2 = sCs[63];  // cs of the last real token (padding adds 0)
        const float keep = exp2f(cl2);
        float wj[MT][4];
#pragma unroll
        for (int jt = 0; jt < MT; ++jt) {
            const f32x4 csq = *reinterpret_cast<const f32x4 *>(&sCs[16 * jt + 4 * grp]);
            const f32x4 dtq = *reinterpret_cast<const f32x4 *>(&sDt[16 * jt + 4 * grp]);
#pragma unroll
            for (int r = 0; r < 4; ++r) wj[jt][r] = exp2f(cl2 - csq[r]) * dtq[r];
        }
        const uint16_t *sBh = reinterpret_cast<const uint16_t *>(sB);
        const float *sBff = reinterpret_cast<const float *>(sBf);
#pragma unroll
        for (int k = 0; k < QW; ++k) {
            const int q = q0 + k;
            // weighted B quad of token tile jt: B[16jt + 4grp + r, 16q + col] w_j
            auto bw = [&](int jt) {
                f32x4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int e = img_idx<QN, F32>(jt, q, col >> 2, 4 * grp + r) * 4 + (col & 3);
                    const float bv = F32 ? sBff[e] : bf16_to_f32(static_cast<short>(sBh[e]));
                    v[r] = bv * wj[jt][r];
                }
                return v;
            };
            f32x4 acc = hq[k] * keep;
            if constexpr (F32) {
#pragma unroll
                for (int jt = 0; jt < MT; ++jt) acc = mma_q32(bw(jt), xquad(jt), acc);
            } else {
                // the weighted B is split into three bf16 terms (the committed state is
                // carried over every later block, so its error must stay at fp32 level),
                // one pair of token tiles at a time
#pragma unroll
                for (int jt = 0; jt < MT; jt += 2) {
                    s16x4 h0, m0, l0;
                    split4x3(bw(jt), h0, m0, l0);
                    if (jt + 1 < MT) {
                        s16x4 h1, m1, l1;
                        split4x3(bw(jt + 1), h1, m1, l1);
                        acc = mma_k32(h0, h1, xq[jt], xq[jt + 1], acc);
                        acc = mma_k32(m0, m1, xq[jt], xq[jt + 1], acc);
                        acc = mma_k32(l0, l1, xq[jt], xq[jt + 1], acc);
                    } else {
                        acc = mma_k16(h0, xq[jt], acc);
                        acc = mma_k16(m0, xq[jt], acc);
                        acc = mma_k16(l0, xq[jt], acc);
                    }
                }
            }
            __builtin_nontemporal_store(acc, reinterpret_cast<f32x4 *>(hs + q * 16 * kP));
            if constexpr (DIR == kCS) hq[k] = acc;   // the next block starts from it
        }
    }

    if constexpr (DIR == kCS) {
        // the next block's first step from the committed state, still in registers: the
        // first group's intra product and skip, every wave's prefix partial product, the
        // partials summed in LDS, y2 stored
        float pre[MT][4], es[MT][4];
        if (part == 0) {
            const float skip = sPar[1] + sPar[2];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                s16x4 mh[MT], ml[MT];
#pragma unroll
                for (int jt = 0; jt < MT; ++jt) {
                    const uint4 v = sM2[(mt * MT + jt) * 64 + lane];
                    mh[jt] = as_s16x4(uint2{v.x, v.y});
                    ml[jt] = as_s16x4(uint2{v.z, v.w});
                }
                f32x4 ai = {0.f, 0.f, 0.f, 0.f};
                ai = mma_quads<MT>(mh, xq2, ai);
                ai = mma_quads<MT>(ml, xq2, ai);
                const f32x4 csq = *reinterpret_cast<const f32x4 *>(&sCs2[16 * mt + 4 * grp]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    pre[mt][r] = ai[r] + skip * xv2[mt][r];
                    es[mt][r] = exp2f(csq[r]);
                }
            }
        }
        f32x4 ap[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) ap[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < QW; k += 2) {
            if (k + 1 < QW) {
                s16x4 h0, l0, h1, l1;
                split4(hq[k], h0, l0);
                split4(hq[k + 1], h1, l1);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const s16x4 c0 = as_s16x4(sC2[img_idx<QN, false>(mt, q0 + k, grp, col)]);
                    const s16x4 c1 = as_s16x4(sC2[img_idx<QN, false>(mt, q0 + k + 1, grp, col)]);
                    ap[mt] = mma_k32(c0, c1, h0, h1, ap[mt]);
                    ap[mt] = mma_k32(c0, c1, l0, l1, ap[mt]);
                }
            } else {
                s16x4 h0, l0;
                split4(hq[k], h0, l0);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const s16x4 c0 = as_s16x4(sC2[img_idx<QN, false>(mt, q0 + k, grp, col)]);
                    ap[mt] = mma_k16(c0, h0, ap[mt]);
                    ap[mt] = mma_k16(c0, l0, ap[mt]);
                }
            }
        }
        if constexpr (NPART > 1) {
            __syncthreads();   // the clean block's partials (if any) have been read
            if (part > 0)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    sRed[(((part - 1) * 4 + pblk) * MT + mt) * 64 + lane] = ap[mt];
            __syncthreads();
            if (part == 0)
#pragma unroll
                for (int pt = 1; pt < NPART; ++pt)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
                        ap[mt] += sRed[(((pt - 1) * 4 + pblk) * MT + mt) * 64 + lane];
        }
        if (part == 0) {
            float *yrow = args.y2 + ((static_cast<int64_t>(b) * L + 4 * grp) * args.nheads + h) * kP + p;
            const int ytok = args.nheads * kP;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (L == LT || 16 * mt + 4 * grp + r < L)
                        __builtin_nontemporal_store(es[mt][r] * ap[mt][r] + pre[mt][r],
                                                    yrow + (16 * mt + r) * ytok);
        }
    }
}

// Zero whole states: grid.y indexes the slot list, grid.x the float4s of a state.
struct ResetArgs {
    float *h_pool;
    int64_t state_elems;
    int64_t first_slot;  // used when use_slots == 0
    int32_t use_slots;
    int32_t slots[BDLM_MAX_SLOT_ROWS];
};

__global__ void __launch_bounds__(256) bdlm_reset_kernel(const ResetArgs a) {
    const int64_t s = a.use_slots ? a.slots[blockIdx.y] : a.first_slot + blockIdx.y;
    f32x4 *dst = reinterpret_cast<f32x4 *>(a.h_pool + s * a.state_elems);
    const int64_t n4 = a.state_elems / 4;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n4;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        dst[i] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Row-major states [n][64][dstate] <-> the pool layout [n][dstate/4][64][4].
// One thread moves one 16-byte quad; i enumerates (state, p, n/4) in row-major order.
__global__ void __launch_bounds__(256)
bdlm_state_permute_kernel(const float *src, float *dst, int64_t nstates, int dstate, int to_pool) {
    const int n4s = dstate / 4;
    const int64_t quads = nstates * kP * n4s;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < quads;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t st = i / (kP * n4s);
        const int rem = static_cast<int>(i - st * kP * n4s);
        const int pp = rem / n4s, n4 = rem - pp * n4s;
        const int64_t rm = (st * kP + pp) * dstate + 4 * n4;
        const int64_t pl = st * kP * dstate + (static_cast<int64_t>(n4) * kP + pp) * 4;
        if (to_pool)
            *reinterpret_cast<f32x4 *>(dst + pl) = *reinterpret_cast<const f32x4 *>(src + rm);
        else
            *reinterpret_cast<f32x4 *>(dst + rm) = *reinterpret_cast<const f32x4 *>(src + pl);
    }
}

// Wave groups per head along dstate.  Measured on MI355X at the 350M layer shape
// (batch 16, 32 heads, dstate 128, L = 32): two groups (8 waves) stream the
// state slightly faster than one; four groups are slower (1024-thread workgroups
// launch more slowly and the reduction barrier lands on the critical path).
template <int LT, int NS>
constexpr int nparts() {
    return (NS / 16) % 2 == 0 ? 2 : 1;
}

template <int LT, int NS, bool F32, bool COMMIT, int DIR>
hipError_t launch_t(const KArgs &k, unsigned grid, hipStream_t s) {
    constexpr int NP = nparts<LT, NS>();
    hipLaunchKernelGGL((bdlm_block_kernel<LT, NS, F32, COMMIT, NP, DIR, false>), dim3(grid),
                       dim3(256 * NP), 0, s, k);
    return hipGetLastError();
}

template <int LT, bool F32, bool COMMIT, int DIR>
hipError_t by_ns(int ns, const KArgs &k, unsigned grid, hipStream_t s) {
    switch (ns) {
        case 16: return launch_t<LT, 16, F32, COMMIT, DIR>(k, grid, s);
        case 32: return launch_t<LT, 32, F32, COMMIT, DIR>(k, grid, s);
        case 64: return launch_t<LT, 64, F32, COMMIT, DIR>(k, grid, s);
        case 128: return launch_t<LT, 128, F32, COMMIT, DIR>(k, grid, s);
        default: return hipErrorInvalidValue;
    }
}

template <bool F32, bool COMMIT, int DIR>
hipError_t by_lt(int L, int ns, const KArgs &k, unsigned grid, hipStream_t s) {
    if (L <= 16) return by_ns<16, F32, COMMIT, DIR>(ns, k, grid, s);
    if (L <= 32) return by_ns<32, F32, COMMIT, DIR>(ns, k, grid, s);
    return by_ns<64, F32, COMMIT, DIR>(ns, k, grid, s);
}

KArgs kargs(const LaunchArgs &a) {
    KArgs k;
    k.x = a.x;
    k.dt = a.dt;
    k.Bm = a.Bm;
    k.Cm = a.Cm;
    k.A = a.A;
    k.D = a.D;
    k.D_rev = a.D_rev;
    k.h_pool = a.h_pool;
    k.y = a.y;
    k.y2 = nullptr;
    k.x2 = k.dt2 = k.Bm2 = k.Cm2 = nullptr;
    k.A2 = nullptr;
    k.conv_w = k.conv_b = k.conv_pool = nullptr;
    k.conv_ch = 0;
    k.xs_b = a.xs_b;
    k.xs_t = a.xs_t;
    k.xs_h = a.xs_h;
    k.dts_b = a.dts_b;
    k.dts_t = a.dts_t;
    k.bcs_b = a.bcs_b;
    k.bcs_t = a.bcs_t;
    k.bcs_g = a.bcs_g;
    k.nheads = a.nheads;
    k.heads_per_group = a.nheads / a.ngroups;
    k.L = a.L;
    const int64_t units = static_cast<int64_t>(a.batch) * a.nheads;
    k.xcd_remap = (units % 8 == 0) ? 1 : 0;
    k.use_slots = a.slots ? 1 : 0;
    for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i) k.slots[i] = (a.slots && i < a.batch) ? a.slots[i] : 0;
    return k;
}

int launch_dir(const LaunchArgs &a, int dir, bool commit, void *stream) {
    const KArgs kn = kargs(a);
    const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(a.batch) * a.nheads);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    switch (dir) {
        case kBoth:
            e = a.bf16 ? (commit ? by_lt<false, true, kBoth>(a.L, a.dstate, kn, grid, s)
                                 : by_lt<false, false, kBoth>(a.L, a.dstate, kn, grid, s))
                       : (commit ? by_lt<true, true, kBoth>(a.L, a.dstate, kn, grid, s)
                                 : by_lt<true, false, kBoth>(a.L, a.dstate, kn, grid, s));
            break;
        case kFwd:
            e = a.bf16 ? (commit ? by_lt<false, true, kFwd>(a.L, a.dstate, kn, grid, s)
                                 : by_lt<false, false, kFwd>(a.L, a.dstate, kn, grid, s))
                       : (commit ? by_lt<true, true, kFwd>(a.L, a.dstate, kn, grid, s)
                                 : by_lt<true, false, kFwd>(a.L, a.dstate, kn, grid, s));
            break;
        default:
            e = commit ? hipErrorInvalidValue
                       : (a.bf16 ? by_lt<false, false, kRev>(a.L, a.dstate, kn, grid, s)
                                 : by_lt<true, false, kRev>(a.L, a.dstate, kn, grid, s));
    }
    return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

}  // namespace

int launch_block(const LaunchArgs &a, bool commit, void *stream) {
    if (a.batch == 0 || a.L == 0) return BDLM_OK;
    return launch_dir(a, kBoth, commit, stream);
}

int launch_block_pair(const LaunchArgs &fwd, const LaunchArgs &rev, bool commit, bool want_y,
                      void *stream) {
    if (fwd.batch == 0 || fwd.L == 0) return BDLM_OK;
    if (!commit && want_y && fwd.bf16 && fwd.L <= 32) {
        // one launch: both branches, each from its own input set
        KArgs k = kargs(fwd);
        k.x2 = rev.x;
        k.dt2 = rev.dt;
        k.Bm2 = rev.Bm;
        k.Cm2 = rev.Cm;
        k.A2 = rev.A;
        k.D_rev = rev.D_rev;
        const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(fwd.batch) * fwd.nheads);
        hipStream_t s = static_cast<hipStream_t>(stream);
        const hipError_t e = fwd.L <= 16 ? by_ns<16, false, false, kSep>(fwd.dstate, k, grid, s)
                                         : by_ns<32, false, false, kSep>(fwd.dstate, k, grid, s);
        return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
    }
    LaunchArgs f = fwd;
    if (!want_y) f.y = nullptr;
    int rc = launch_dir(f, kFwd, commit, stream);
    if (rc != BDLM_OK || !want_y) return rc;
    return launch_dir(rev, kRev, false, stream);
}

int launch_commit_step(const LaunchArgs &clean, const LaunchArgs &next, float *y_next,
                       void *stream) {
    if (clean.batch == 0) return BDLM_OK;
    if (clean.L == 0) {   // nothing to commit: the next block's step alone
        LaunchArgs n = next;
        n.y = y_next;
        return launch_block(n, false, stream);
    }
    if (clean.bf16 && clean.L <= 32) {
        KArgs k = kargs(clean);
        k.x2 = next.x;
        k.dt2 = next.dt;
        k.Bm2 = next.Bm;
        k.Cm2 = next.Cm;
        k.y2 = y_next;
        const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(clean.batch) * clean.nheads);
        hipStream_t s = static_cast<hipStream_t>(stream);
        const hipError_t e = clean.L <= 16 ? by_ns<16, false, true, kCS>(clean.dstate, k, grid, s)
                                           : by_ns<32, false, true, kCS>(clean.dstate, k, grid, s);
        return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
    }
    // otherwise the commit, then the step, as two launches on the stream
    int rc = launch_block(clean, true, stream);
    if (rc != BDLM_OK) return rc;
    LaunchArgs n = next;
    n.y = y_next;
    return launch_block(n, false, stream);
}

template <int LT, bool COMMIT, int DIR>
hipError_t conv_by_ns(int ns, const KArgs &k, unsigned grid, hipStream_t s) {
    switch (ns) {
#define BDLM_CONV_NS(N)                                                                          \
    case N: {                                                                                    \
        constexpr int NP = nparts<LT, N>();                                                      \
        hipLaunchKernelGGL((bdlm_block_kernel<LT, N, true, COMMIT, NP, DIR, true>), dim3(grid),   \
                           dim3(256 * NP), 0, s, k);                                             \
        return hipGetLastError();                                                                \
    }
        BDLM_CONV_NS(16)
        BDLM_CONV_NS(32)
        BDLM_CONV_NS(64)
        BDLM_CONV_NS(128)
#undef BDLM_CONV_NS
        default: return hipErrorInvalidValue;
    }
}

int launch_conv_fused(const LaunchArgs &a, const float *w, const float *bias, const float *conv_pool,
                      bool commit, bool want_y, void *stream) {
    if (a.batch == 0 || a.L == 0) return BDLM_OK;
    KArgs k = kargs(a);
    k.conv_w = w;
    k.conv_b = bias;
    k.conv_pool = conv_pool;
    k.conv_ch = a.nheads * kP + 2 * a.ngroups * a.dstate;
    const unsigned grid = static_cast<unsigned>(static_cast<int64_t>(a.batch) * a.nheads);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (want_y) {
        // one launch: both convolutions staged side by side (the forward one as the first
        // input set, the reverse one as the second, same dt and A), both branches' intra
        // products, the prefix term, a commit's state update from the forward set
        k.dt2 = a.dt;
        k.A2 = a.A;
        if (a.L <= 16)
            e = commit ? conv_by_ns<16, true, kSep>(a.dstate, k, grid, s) : conv_by_ns<16, false, kSep>(a.dstate, k, grid, s);
        else
            e = commit ? conv_by_ns<32, true, kSep>(a.dstate, k, grid, s) : conv_by_ns<32, false, kSep>(a.dstate, k, grid, s);
        return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
    }
    // a commit without outputs: the forward convolution and the state update alone
    KArgs f = k;
    f.y = nullptr;
    e = a.L <= 16 ? conv_by_ns<16, true, kFwd>(a.dstate, f, grid, s) : conv_by_ns<32, true, kFwd>(a.dstate, f, grid, s);
    return e == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

int launch_state_permute(const float *src, float *dst, int64_t nstates, int64_t dstate,
                         bool to_pool, void *stream) {
    const int64_t quads = nstates * kP * (dstate / 4);
    if (quads == 0) return BDLM_OK;
    const int64_t want = (quads + 255) / 256;
    const unsigned grid = static_cast<unsigned>(want < 8192 ? want : 8192);
    hipLaunchKernelGGL(bdlm_state_permute_kernel, dim3(grid), dim3(256), 0,
                       static_cast<hipStream_t>(stream), src, dst, nstates,
                       static_cast<int>(dstate), to_pool ? 1 : 0);
    return hipGetLastError() == hipSuccess ? BDLM_OK : BDLM_E_LAUNCH;
}

int launch_reset(float *h_pool, int64_t nslots, int64_t state_elems, const int32_t *slots,
                 int64_t nreset, void *stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t n4 = state_elems / 4;
    const unsigned gx = static_cast<unsigned>(n4 < 256 * 64 ? (n4 + 255) / 256 : 64);
    const int64_t count = slots ? nreset : nslots;
    for (int64_t done = 0; done < count; done += BDLM_MAX_SLOT_ROWS) {
        const int64_t chunk = count - done < BDLM_MAX_SLOT_ROWS ? count - done : BDLM_MAX_SLOT_ROWS;
        ResetArgs r;
        r.h_pool = h_pool;
        r.state_elems = state_elems;
        r.first_slot = done;
        r.use_slots = slots ? 1 : 0;
        for (int i = 0; i < BDLM_MAX_SLOT_ROWS; ++i) r.slots[i] = (slots && i < chunk) ? slots[done + i] : 0;
        hipLaunchKernelGGL(bdlm_reset_kernel, dim3(gx > 0 ? gx : 1, static_cast<unsigned>(chunk)),
                           dim3(256), 0, s, r);
        if (hipGetLastError() != hipSuccess) return BDLM_E_LAUNCH;
    }
    return BDLM_OK;
}

}  // namespace bdlm
